// C ABI of libps: validation, the error model, per-call metadata upload and
// the layer executor that sequences the kernels of one prefill, decode or
// mixed step.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <cmath>
#include <cstring>
#include <initializer_list>
#include <new>
#include <string>
#include <thread>
#include <vector>

#include "../../include/ps.h"
#include "admission.h"
#include "control.h"
#include "common.h"
#include "kv_pool.h"
#include "launch.h"

using namespace ps;

// ------------------------------------------------------------------ errors
namespace {
thread_local std::string g_err;

ps_status fail(ps_status code, const std::string& msg) {
  g_err = msg;
  return code;
}

#define PS_TRY try {
#define PS_CATCH                                                   \
  }                                                                \
  catch (const std::bad_alloc&) {                                  \
    return fail(PS_E_INVALID, "host allocation failed");           \
  }                                                                \
  catch (...) {                                                    \
    return fail(PS_E_INVALID, "internal error");                   \
  }

// Device buffers are accessed with 16-byte vector loads and stores.
ps_status check_aligned(std::initializer_list<const void*> ptrs) {
  for (const void* p : ptrs)
    if ((uintptr_t)p & 15) return fail(PS_E_INVALID, "device buffers must be 16-byte aligned");
  return PS_OK;
}

ps_status hip_fail(hipError_t e, const char* what) {
  return fail(PS_E_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

int elt_bytes(int dt) { return dt == PS_BF16 ? 2 : 4; }

// Field by field: ps_layer_cfg has tail padding after `dtype`, which a
// caller's separately built configurations need not agree on.
bool same_cfg(const ps_layer_cfg& a, const ps_layer_cfg& b) {
  return a.hidden == b.hidden && a.n_q_heads == b.n_q_heads && a.n_kv_heads == b.n_kv_heads &&
         a.head_dim == b.head_dim && a.ffn == b.ffn && a.rms_eps == b.rms_eps && a.rope_theta == b.rope_theta &&
         a.dtype == b.dtype;
}

ps_status check_cfg(const ps_layer_cfg* c) {
  if (!c) return fail(PS_E_INVALID, "null config");
  if (c->dtype != PS_F32 && c->dtype != PS_BF16) return fail(PS_E_INVALID, "dtype must be PS_F32 or PS_BF16");
  if (c->hidden <= 0 || c->n_q_heads <= 0 || c->n_kv_heads <= 0 || c->head_dim <= 0 || c->ffn <= 0)
    return fail(PS_E_INVALID, "non-positive dimension");
  if (c->n_q_heads % c->n_kv_heads) return fail(PS_E_INVALID, "n_kv_heads must divide n_q_heads");
  if (c->head_dim % 2 || c->head_dim > 128) return fail(PS_E_UNSUPPORTED, "head_dim must be even and <= 128");
  if (c->ffn % PS_GATE_UP_BLOCK) return fail(PS_E_UNSUPPORTED, "ffn must be a multiple of PS_GATE_UP_BLOCK");
  if (!(c->rms_eps >= 0.f) || !(c->rope_theta > 0.0)) return fail(PS_E_INVALID, "bad eps or rope_theta");
  return PS_OK;
}

// Pinned host staging ring for per-call metadata. A slot is reused only
// after the upload kernel that last read it has run: every workgroup of that
// kernel stores the upload's tag into a word of pinned host memory once its
// reads are done, and the host waits for those words (no event sits in the
// caller's stream, so nothing there depends on which streams the calls use).
struct Staging {
  static constexpr int kSlots = 4;
  void* host[kSlots] = {};
  void* mapped[kSlots] = {};  // device-side address of host[s]
  size_t cap[kSlots] = {};
  uint32_t* done = nullptr;  // kSlots x kUploadMaxBlocks words written by the upload kernel
  uint32_t* done_mapped = nullptr;
  uint32_t tag[kSlots] = {};  // tag of the slot's last upload
  int blocks[kSlots] = {};    // its workgroups; 0 = nothing outstanding
  uint32_t last_tag = 0;
  int next = 0;

  // Waits until slot s's last upload has read the slot; false after
  // `limit` with the upload still outstanding.
  bool wait(int s, std::chrono::seconds limit) {
    if (!blocks[s]) return true;
    const volatile uint32_t* d = done + (size_t)s * kUploadMaxBlocks;
    const auto t0 = std::chrono::steady_clock::now();
    for (int b = 0; b < blocks[s]; ++b)
      for (unsigned spin = 0; d[b] != tag[s]; ++spin) {
        std::this_thread::yield();
        if ((spin & 4095) == 4095 && std::chrono::steady_clock::now() - t0 > limit) return false;
      }
    std::atomic_thread_fence(std::memory_order_acquire);
    blocks[s] = 0;
    return true;
  }
  ~Staging() {
    bool drained = true;
    for (int s = 0; s < kSlots; ++s) drained = wait(s, std::chrono::seconds(10)) && drained;
    if (!drained) return;  // the device may still read the ring: leave it allocated
    for (int s = 0; s < kSlots; ++s)
      if (host[s]) (void)hipHostFree(host[s]);
    if (done) (void)hipHostFree(done);
  }
  // Returns the slot index or -1 (g_err set).
  int acquire(size_t bytes, void** out) {
    hipError_t e;
    if (!done) {
      const size_t nb = sizeof(uint32_t) * kSlots * kUploadMaxBlocks;
      if ((e = hipHostMalloc((void**)&done, nb, hipHostMallocMapped | hipHostMallocCoherent)) != hipSuccess)
        return (done = nullptr, hip_fail(e, "staging hipHostMalloc"), -1);
      std::memset(done, 0, nb);
      if ((e = hipHostGetDevicePointer((void**)&done_mapped, done, 0)) != hipSuccess)
        return (hip_fail(e, "staging device pointer"), -1);
    }
    const int s = next;
    if (!wait(s, std::chrono::seconds(60)))
      return (fail(PS_E_HIP, "staging wait: the upload that last used the slot has not run after 60 s"), -1);
    if (cap[s] < bytes) {
      if (!grow(s, bytes)) return -1;
      // slots never used yet are allocated now too, so that a loop of calls
      // does not pay a pinned allocation in each of its first kSlots calls
      for (int j = 0; j < kSlots; ++j)
        if (!host[j] && !grow(j, bytes)) return -1;
    }
    *out = host[s];
    return s;
  }
  // (Re)allocates slot j, which no outstanding upload reads, for `bytes`.
  bool grow(int j, size_t bytes) {
    if (host[j]) (void)hipHostFree(host[j]);
    host[j] = mapped[j] = nullptr;
    cap[j] = 0;
    const size_t nb = align_up(std::max<size_t>(bytes, 1 << 16), 1 << 16);
    hipError_t e;
    // coherent (uncached on the device): the upload kernel reads what the
    // host wrote just before the launch
    if ((e = hipHostMalloc(&host[j], nb, hipHostMallocMapped | hipHostMallocCoherent)) != hipSuccess)
      return (host[j] = nullptr, hip_fail(e, "staging hipHostMalloc"), false);
    if ((e = hipHostGetDevicePointer(&mapped[j], host[j], 0)) != hipSuccess)
      return (hip_fail(e, "staging device pointer"), false);
    cap[j] = nb;
    return true;
  }
  // The upload of the slot's first `bytes`, rounded up to 16, to `dev`
  // (slots are acquired for the 256-aligned metadata size, and the
  // destination always has that much room). Marks the slot as read by that
  // upload: the caller enqueues the job (launch_upload, or a kernel that
  // carries it) before it touches the ring again. The ring advances only
  // here, so a slot acquired by a call that then failed is acquired again.
  ps_status prepare(int s, void* dev, size_t bytes, UploadJob* job) {
    const uint32_t t = last_tag + 1 ? last_tag + 1 : 1;  // 0 is the words' initial value
    if (!make_upload_job(mapped[s], dev, align_up(bytes, 16), done_mapped + (size_t)s * kUploadMaxBlocks, t, job))
      return fail(PS_E_INVALID, "metadata upload size");
    last_tag = t;
    tag[s] = t;
    blocks[s] = job->blocks;
    next = (s + 1) % kSlots;
    return PS_OK;
  }
  // prepare + the upload as its own kernel on `st`.
  ps_status submit(int s, void* dev, size_t bytes, hipStream_t st) {
    UploadJob j;
    if (ps_status rc = prepare(s, dev, bytes, &j)) return rc;
    launch_upload(j, st);
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? PS_OK : hip_fail(e, "metadata upload");
  }
};

// Per-call metadata, assembled on the host and uploaded in one copy to the
// head of the caller's workspace.
struct Meta {
  std::vector<uint8_t> buf;
  size_t add(const void* p, size_t bytes) {
    size_t off = align_up(buf.size(), 256);
    buf.resize(off + bytes);
    if (bytes) std::memcpy(buf.data() + off, p, bytes);
    return off;
  }
  size_t size() const { return align_up(buf.size(), 256); }
};
}  // namespace

// Host record of the last ps_op_decode_plan on a handle: where its work
// list sits in the caller's workspace and the pool state it was made for.
struct DecodeAttnPlan {
  const void* ws = nullptr;
  size_t ws_need = 0;
  uint64_t gen = 0;
  int32_t n_seqs = 0, n_items = 0;
  size_t o_si = 0, o_bt = 0, o_di = 0, o_pb = 0, o_pc = 0, off_po = 0, off_pml = 0;
};

struct ps_kv {
  ps_layer_cfg cfg;
  int32_t n_layers;
  void* pool;
  size_t layer_elts;  // elements per layer
  KvPool meta;
  Staging staging;
  DecodeAttnPlan dplan;
  ps_kv(const ps_layer_cfg& c, int32_t nl, int32_t np, int32_t ms, int32_t mp, void* p, uint64_t seed)
      : cfg(c), n_layers(nl), pool(p),
        layer_elts((size_t)np * c.n_kv_heads * 2 * PS_PAGE_TOKENS * c.head_dim), meta(np, ms, mp, seed) {}
  void* layer_base(int layer) const {
    return (char*)pool + (size_t)layer * layer_elts * elt_bytes(cfg.dtype);
  }
};

// A second stream on the caller's device (default priority, non-blocking)
// and the events that fork a mixed step's work onto it and join it back
// inside one call. Created on first use; a layer handle is driven by one host
// thread at a time.
struct AuxStream {
  static constexpr int kEvents = 2;
  int dev = -1;
  hipStream_t s = nullptr;
  hipEvent_t ev[kEvents] = {};
  AuxStream() = default;
  AuxStream(const AuxStream&) = delete;
  AuxStream& operator=(const AuxStream&) = delete;
  ~AuxStream() {
    for (hipEvent_t& e : ev)
      if (e) (void)hipEventDestroy(e);
    if (s) (void)hipStreamDestroy(s);
  }
  // *out = this, ready for work forked from `caller`, or nullptr when the
  // caller's stream is not on the current device or the stream was made
  // for another device (the call then runs on the caller's stream alone).
  ps_status get(hipStream_t caller, AuxStream** out) {
    *out = nullptr;
    int cur = 0, sdev = 0;
    if (hipError_t e = hipGetDevice(&cur)) return hip_fail(e, "current device");
    if (caller) {
      if (hipError_t e = hipStreamGetDevice(caller, &sdev)) return hip_fail(e, "stream device");
    } else {
      sdev = cur;
    }
    if (sdev != cur || (dev >= 0 && dev != cur)) return PS_OK;
    if (dev < 0) {
      hipStream_t ns = nullptr;
      hipEvent_t ne[kEvents] = {};
      hipError_t e = hipStreamCreateWithFlags(&ns, hipStreamNonBlocking);
      for (int i = 0; i < kEvents && e == hipSuccess; ++i) e = hipEventCreateWithFlags(&ne[i], hipEventDisableTiming);
      if (e != hipSuccess) {
        for (hipEvent_t x : ne)
          if (x) (void)hipEventDestroy(x);
        if (ns) (void)hipStreamDestroy(ns);
        return hip_fail(e, "auxiliary stream and its events");
      }
      s = ns;
      for (int i = 0; i < kEvents; ++i) ev[i] = ne[i];
      dev = cur;
    }
    *out = this;
    return PS_OK;
  }
};

struct ps_layer {
  ps_layer_cfg cfg;
  AuxStream aux;
};

struct ps_model {
  ps_layer_cfg cfg;
  int32_t n_layers = 0, vocab = 0;
  const void* embed = nullptr;
  const void* final_norm = nullptr;
  const void* lm_head = nullptr;
  std::vector<ps_layer_w> layers;
};

// ------------------------------------------------------------------ misc
extern "C" const char* ps_last_error(void) { return g_err.c_str(); }
extern "C" const char* ps_version(void) { return "libps 0.2.0 gfx950"; }

extern "C" ps_status ps_get_device_info(int32_t device, ps_device_info* out) {
  PS_TRY
  if (!out) return fail(PS_E_INVALID, "null out");
  hipDeviceProp_t p;
  if (hipError_t e = hipGetDeviceProperties(&p, device)) return hip_fail(e, "hipGetDeviceProperties");
  std::memset(out, 0, sizeof(*out));
  out->compute_units = p.multiProcessorCount;
  out->clock_khz = p.clockRate;
  out->memory_clock_khz = p.memoryClockRate;
  out->memory_bus_bits = p.memoryBusWidth;
  out->total_memory = (int64_t)p.totalGlobalMem;
  out->l2_bytes = p.l2CacheSize;
  out->lds_bytes_per_block = (int32_t)p.sharedMemPerBlock;
  std::strncpy(out->arch, p.gcnArchName, sizeof(out->arch) - 1);
  return PS_OK;
  PS_CATCH
}

extern "C" ps_status ps_pack_gate_up(const void* wg, const void* wu, int32_t F, int32_t d, int32_t eb, void* out) {
  PS_TRY
  if (!wg || !wu || !out || F <= 0 || d <= 0 || (eb != 2 && eb != 4)) return fail(PS_E_INVALID, "bad arguments");
  if (F % PS_GATE_UP_BLOCK) return fail(PS_E_INVALID, "F must be a multiple of PS_GATE_UP_BLOCK");
  const size_t row = (size_t)d * eb;
  for (int32_t blk = 0; blk < F / PS_GATE_UP_BLOCK; ++blk)
    for (int32_t r = 0; r < PS_GATE_UP_BLOCK; ++r) {
      const size_t src = (size_t)(blk * PS_GATE_UP_BLOCK + r) * row;
      std::memcpy((char*)out + (size_t)(2 * blk * PS_GATE_UP_BLOCK + r) * row, (const char*)wg + src, row);
      std::memcpy((char*)out + (size_t)((2 * blk + 1) * PS_GATE_UP_BLOCK + r) * row, (const char*)wu + src, row);
    }
  return PS_OK;
  PS_CATCH
}

extern "C" size_t ps_tiled_weight_elems(int32_t N, int32_t K) {
  if (N <= 0 || K <= 0) return 0;
  return (size_t)tiled_weight_elems(N, K);
}

extern "C" ps_status ps_tile_weight(const void* w, int32_t N, int32_t K, int32_t eb, void* out) {
  PS_TRY
  if (!w || !out || N <= 0 || K <= 0 || (eb != 2 && eb != 4)) return fail(PS_E_INVALID, "bad arguments");
  const long kt = (K + kWTile - 1) / kWTile, nt = (N + kWTile - 1) / kWTile;
  std::memset(out, 0, (size_t)tiled_weight_elems(N, K) * eb);
  for (long i = 0; i < nt; ++i)
    for (long j = 0; j < kt; ++j) {
      const long cols = std::min<long>(kWTile, K - j * kWTile);
      char* tile = (char*)out + (size_t)(i * kt + j) * kWTileElts * eb;
      for (long r = 0; r < kWTile && i * kWTile + r < N; ++r)
        std::memcpy(tile + (size_t)r * kWTile * eb, (const char*)w + ((size_t)(i * kWTile + r) * K + j * kWTile) * eb,
                    (size_t)cols * eb);
    }
  return PS_OK;
  PS_CATCH
}

// ------------------------------------------------------------------ KV pool
extern "C" size_t ps_kv_pool_bytes(const ps_layer_cfg* c, int32_t n_layers, int32_t n_pages) {
  if (!c || n_layers <= 0 || n_pages <= 0) return 0;
  return (size_t)n_layers * n_pages * c->n_kv_heads * 2 * PS_PAGE_TOKENS * c->head_dim * elt_bytes(c->dtype);
}

extern "C" ps_status ps_kv_create(const ps_layer_cfg* c, int32_t n_layers, int32_t n_pages, int32_t max_seqs,
                                  int32_t max_pages_per_seq, void* pool, uint64_t seed, ps_kv** out) {
  PS_TRY
  if (ps_status rc = check_cfg(c)) return rc;
  if (!out) return fail(PS_E_INVALID, "null out");
  if (n_layers <= 0 || n_pages <= 0 || max_seqs <= 0 || max_pages_per_seq <= 0)
    return fail(PS_E_INVALID, "non-positive pool size");
  if (!pool) return fail(PS_E_INVALID, "null pool");
  if (ps_status rc = check_aligned({pool})) return rc;
  *out = new ps_kv(*c, n_layers, n_pages, max_seqs, max_pages_per_seq, pool, seed);
  return PS_OK;
  PS_CATCH
}

extern "C" ps_status ps_kv_destroy(ps_kv* kv) {
  PS_TRY
  delete kv;
  return PS_OK;
  PS_CATCH
}

#define CHECK_KV(kv) \
  if (!(kv)) return fail(PS_E_INVALID, "null kv handle");

extern "C" ps_status ps_kv_seq_open(ps_kv* kv, int32_t* seq) {
  PS_TRY CHECK_KV(kv);
  if (!seq) return fail(PS_E_INVALID, "null seq");
  std::string e;
  if (int rc = kv->meta.open(seq, e)) return fail(rc, e);
  return PS_OK;
  PS_CATCH
}
extern "C" ps_status ps_kv_alloc(ps_kv* kv, int32_t seq, int32_t n) {
  PS_TRY CHECK_KV(kv);
  std::string e;
  if (int rc = kv->meta.reserve(seq, n, e)) return fail(rc, e);
  return PS_OK;
  PS_CATCH
}
extern "C" ps_status ps_kv_commit(ps_kv* kv, int32_t n, const int32_t* seqs, const int32_t* n_tok) {
  PS_TRY CHECK_KV(kv);
  std::string e;
  if (int rc = kv->meta.commit(n, seqs, n_tok, e)) return fail(rc, e);
  return PS_OK;
  PS_CATCH
}
extern "C" ps_status ps_kv_truncate(ps_kv* kv, int32_t seq, int32_t new_len) {
  PS_TRY CHECK_KV(kv);
  std::string e;
  if (int rc = kv->meta.truncate(seq, new_len, e)) return fail(rc, e);
  return PS_OK;
  PS_CATCH
}
extern "C" ps_status ps_kv_free(ps_kv* kv, int32_t seq) {
  PS_TRY CHECK_KV(kv);
  std::string e;
  if (int rc = kv->meta.release(seq, e)) return fail(rc, e);
  return PS_OK;
  PS_CATCH
}
extern "C" ps_status ps_kv_seq_len(const ps_kv* kv, int32_t seq, int32_t* len) {
  PS_TRY CHECK_KV(kv);
  std::string e;
  if (!len) return fail(PS_E_INVALID, "null len");
  if (int rc = kv->meta.check_open(seq, e)) return fail(rc, e);
  *len = kv->meta.seq(seq).len;
  return PS_OK;
  PS_CATCH
}
extern "C" ps_status ps_kv_capacity(const ps_kv* kv, int32_t seq, int32_t* tokens) {
  PS_TRY CHECK_KV(kv);
  std::string e;
  if (!tokens) return fail(PS_E_INVALID, "null tokens");
  if (int rc = kv->meta.check_open(seq, e)) return fail(rc, e);
  *tokens = kv->meta.capacity(seq);
  return PS_OK;
  PS_CATCH
}
extern "C" ps_status ps_kv_free_pages(const ps_kv* kv, int32_t* n) {
  PS_TRY CHECK_KV(kv);
  if (!n) return fail(PS_E_INVALID, "null n");
  *n = kv->meta.free_pages();
  return PS_OK;
  PS_CATCH
}
extern "C" ps_status ps_kv_block_table(const ps_kv* kv, int32_t seq, int32_t* pages, int32_t cap, int32_t* n) {
  PS_TRY CHECK_KV(kv);
  std::string e;
  if (!n) return fail(PS_E_INVALID, "null n");
  if (int rc = kv->meta.check_open(seq, e)) return fail(rc, e);
  const auto& p = kv->meta.seq(seq).pages;
  *n = (int32_t)p.size();
  if (pages) std::memcpy(pages, p.data(), sizeof(int32_t) * std::min<size_t>(p.size(), cap > 0 ? cap : 0));
  return PS_OK;
  PS_CATCH
}

// ------------------------------------------------------------ call planning
namespace {

// Sequences of one call: `groups` is the list of (seq, n_new) in row order.
struct CallSeqs {
  std::vector<SeqInfo> si;
  std::vector<int32_t> bt;  // compact block table
  int32_t rows = 0;
};

ps_status plan_seqs(const ps_kv* kv, int n, const int32_t* seqs, const int32_t* n_tok, int32_t fixed_n,
                    CallSeqs& cs) {
  if (n < 0 || (n > 0 && !seqs)) return fail(PS_E_INVALID, "bad sequence list");
  if (fixed_n < 0 && n > 0 && !n_tok) return fail(PS_E_INVALID, "null n_tok");
  std::string e;
  for (int i = 0; i < n; ++i) {
    const int32_t s = seqs[i];
    const int32_t nn = fixed_n >= 0 ? fixed_n : n_tok[i];
    if (nn <= 0) return fail(PS_E_INVALID, "every sequence needs at least one new token");
    if (int rc = kv->meta.check_writable(s, nn, e)) return fail(rc, e);
    for (int j = 0; j < i; ++j)
      if (seqs[j] == s) return fail(PS_E_INVALID, "sequence listed twice in one call");
    const KvSeq& q = kv->meta.seq(s);
    SeqInfo inf;
    inf.kv_before = q.len;
    inf.n_new = nn;
    inf.row_start = cs.rows;
    inf.bt_off = (int32_t)cs.bt.size();
    const int32_t pages = (q.len + nn + PS_PAGE_TOKENS - 1) / PS_PAGE_TOKENS;
    cs.bt.insert(cs.bt.end(), q.pages.begin(), q.pages.begin() + pages);
    cs.si.push_back(inf);
    cs.rows += nn;
  }
  return PS_OK;
}

struct DecodePlan {
  std::vector<DecodeItem> items;
  std::vector<int32_t> part_begin, part_count;
  int32_t n_parts = 0;
};

int32_t choose_split_pages(const std::vector<SeqInfo>& si, size_t first, int n_kv, int phase) {
  (void)phase;
  long total = 0;
  for (size_t b = first; b < si.size(); ++b) total += (si[b].kv_before + si[b].n_new + 15) / 16;
  // At most about 1024 workgroups over the chip: two full rounds of the 512
  // that fit at two per CU, at least 8 pages per split, a multiple of 4 (the
  // four waves of a workgroup walk pages w, w + 4, ...). Measured over split
  // sizes on the 8B decode and think and the 70B decode workloads: every
  // workgroup pays a ramp-up (its first pages' latency) and a merge, so
  // fewer, longer splits stream faster down to ~1000 workgroups (3072: 5-10%
  // slower), and a plan that spills a few items into a third round pays for
  // that round (think batch: 1152 workgroups 285 us, 1000 workgroups 274 us).
  // So the split is the smallest that keeps the grid within two rounds,
  // where one exists; a batch of more sequences than two rounds hold gets
  // one split per sequence.
  auto n_items = [&](long spl) {
    long n = 0;
    for (size_t b = first; b < si.size(); ++b) n += ((si[b].kv_before + si[b].n_new + 15) / 16 + spl - 1) / spl;
    return n;
  };
  long max_pages = 8;
  for (size_t b = first; b < si.size(); ++b) max_pages = std::max<long>(max_pages, (si[b].kv_before + si[b].n_new + 15) / 16);
  const long target_items = std::max(1, 1024 / std::max(1, n_kv));
  long sp = std::max<long>((total + target_items - 1) / target_items, 8);
  sp = (sp + 3) / 4 * 4;
  if (n_items(sp) > target_items) {  // smallest multiple of 4 in (sp, max_pages] that fits: n_items falls as sp grows
    long lo = sp / 4, hi = (max_pages + 3) / 4;
    while (lo + 1 < hi) {
      const long mid = (lo + hi) / 2;
      if (n_items(4 * mid) <= target_items) hi = mid;
      else lo = mid;
    }
    sp = 4 * hi;
  }
  // the work-item index is a grid y coordinate (at most 65535): widen the
  // splits until the items fit (a batch of more sequences than that is
  // rejected by the launcher)
  while (n_items(sp) > kMaxDecodeItems && sp < (1L << 24)) sp *= 2;
  return (int32_t)sp;
}

DecodePlan plan_decode(const std::vector<SeqInfo>& si, size_t first, int32_t split_pages) {
  DecodePlan p;
  for (size_t b = first; b < si.size(); ++b) {
    const int32_t np = (si[b].kv_before + si[b].n_new + 15) / 16;
    const int32_t ns = (np + split_pages - 1) / split_pages;
    p.part_begin.push_back(p.n_parts);
    p.part_count.push_back(ns);
    // ns splits of at most split_pages pages, as even as possible (sizes
    // differ by at most one page), so no short remainder split trails
    for (int32_t k = 0; k < ns; ++k) {
      DecodeItem it;
      it.b = (int32_t)(b - first);
      it.page_begin = (int32_t)((long)k * np / ns);
      it.page_end = (int32_t)((long)(k + 1) * np / ns);
      it.part = p.n_parts + k;
      p.items.push_back(it);
    }
    p.n_parts += ns;
  }
  // longest splits first
  std::stable_sort(p.items.begin(), p.items.end(), [](const DecodeItem& a, const DecodeItem& c) {
    return (a.page_end - a.page_begin) > (c.page_end - c.page_begin);
  });
  return p;
}

std::vector<PrefillItem> plan_prefill(const std::vector<SeqInfo>& si, size_t count) {
  std::vector<PrefillItem> it;
  for (size_t b = 0; b < count; ++b)
    for (int32_t q0 = 0; q0 < si[b].n_new; q0 += fa_query_tile()) it.push_back(PrefillItem{(int32_t)b, q0});
  // most keys first (causal imbalance)
  std::stable_sort(it.begin(), it.end(), [&](const PrefillItem& a, const PrefillItem& c) {
    return si[a.b].kv_before + a.q_begin > si[c.b].kv_before + c.q_begin;
  });
  return it;
}

bool use_mfma_attn(const ps_layer_cfg& c) { return c.dtype == PS_BF16 && c.head_dim == 128; }
int group_of(const ps_layer_cfg& c) { return c.n_q_heads / c.n_kv_heads; }
bool fa_ok(const ps_layer_cfg& c) { return use_mfma_attn(c) && group_of(c) % 4 == 0 && group_of(c) <= 64; }
bool dec_ok(const ps_layer_cfg& c) {
  const int g = group_of(c);
  return use_mfma_attn(c) && (g == 1 || g == 2 || g == 4 || g == 8 || g == 16);
}

std::vector<double> inv_freq(const ps_layer_cfg& c) {
  std::vector<double> f(c.head_dim / 2);
  for (int j = 0; j < c.head_dim / 2; ++j) f[j] = std::pow(c.rope_theta, -2.0 * j / c.head_dim);
  return f;
}

// Workspace carve-out for a layer call (after the metadata region).
struct WsLayout {
  size_t xn, qkv, qr, o, h, m, gemm, gemm_b, apart_o, apart_ml, total;
};

WsLayout layout(const ps_layer_cfg& c, size_t meta_bytes, int32_t rows, int32_t n_parts_max) {
  const size_t eb = elt_bytes(c.dtype);
  const size_t d = c.hidden, dq = (size_t)c.n_q_heads * c.head_dim, dkv = (size_t)c.n_kv_heads * c.head_dim;
  WsLayout L;
  size_t off = align_up(meta_bytes, 256);
  auto take = [&](size_t bytes) {
    size_t o = off;
    off = align_up(off + bytes, 256);
    return o;
  };
  L.xn = take(rows * d * eb);
  L.qkv = take(rows * (dq + 2 * dkv) * eb);
  L.qr = take(rows * dq * eb);
  L.o = take(rows * dq * eb);
  L.h = take(rows * d * 4);
  L.m = take(rows * (size_t)c.ffn * eb);
  // split-K partials of the decode-sized GEMMs, sized for min(rows, 64)
  // rows so that a bound taken for more rows also covers smaller calls
  size_t g = 0;
  const int gm = std::min(rows, 64);
  if (gm > 0) {
    g = std::max(g, gemm_workspace_bytes(c.dtype, gm, (int)(dq + 2 * dkv), (int)d));
    g = std::max(g, gemm_workspace_bytes(c.dtype, gm, (int)d, (int)dq));
    g = std::max(g, gemm_workspace_bytes(c.dtype, gm, 2 * c.ffn, (int)d));
    g = std::max(g, gemm_workspace_bytes(c.dtype, gm, (int)d, c.ffn));
  }
  // K-split partials of the tile-path O and down GEMMs, for any row count
  // up to `rows` (a call's chunk rows included)
  if (c.dtype == PS_BF16 && rows > 0) {
    g = std::max(g, gemm_tile_partials_bound(rows, (int)d, (int)dq));
    g = std::max(g, gemm_tile_partials_bound(rows, (int)d, c.ffn));
  }
  L.gemm = take(g);
  // the decode rows' O, SwiGLU and down partials when they run on the
  // second stream beside the chunk rows
  size_t gb = 0;
  if (gm > 0) {
    gb = std::max(gb, gemm_workspace_bytes(c.dtype, gm, (int)d, (int)dq));
    gb = std::max(gb, gemm_workspace_bytes(c.dtype, gm, 2 * c.ffn, (int)d));
    gb = std::max(gb, gemm_workspace_bytes(c.dtype, gm, (int)d, c.ffn));
  }
  L.gemm_b = take(gb);
  L.apart_o = take((size_t)n_parts_max * dq * 4);
  L.apart_ml = take((size_t)n_parts_max * c.n_q_heads * 2 * 4);
  L.total = off;
  return L;
}

size_t meta_bound(const ps_layer_cfg& c, int32_t max_rows, int32_t max_seqs, int32_t max_pages) {
  size_t b = 0;
  b += align_up(sizeof(SeqInfo) * max_seqs, 256);
  b += align_up(4ull * max_seqs * max_pages, 256);
  b += align_up(8ull * c.head_dim / 2, 256);
  const size_t parts = (size_t)max_seqs * ((max_pages + 7) / 8);
  b += align_up(sizeof(DecodeItem) * parts, 256) + 2 * align_up(4ull * max_seqs, 256);
  b += align_up(sizeof(PrefillItem) * ((size_t)max_rows / 32 + max_seqs), 256);
  return b + 256;
}

ps_status check_ws(const void* ws, size_t have, size_t need) {
  if (!ws) return fail(PS_E_INVALID, "null workspace");
  if ((uintptr_t)ws & 15) return fail(PS_E_INVALID, "workspace must be 16-byte aligned");
  if (have < need)
    return fail(PS_E_INVALID, "workspace too small: " + std::to_string(have) + " < " + std::to_string(need));
  return PS_OK;
}

ps_status check_layer(const ps_kv* kv, int layer) {
  if (layer < 0 || layer >= kv->n_layers) return fail(PS_E_INVALID, "layer index out of range");
  return PS_OK;
}

ps_status last_launch_error() {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "kernel launch");
  return PS_OK;
}

}  // namespace

// ------------------------------------------------------------ KV device ops
extern "C" ps_status ps_kv_append(ps_kv* kv, int32_t layer, int32_t n_seqs, const int32_t* seqs,
                                  const int32_t* n_tok, const void* k, const void* v, void* ws, size_t ws_bytes,
                                  void* stream) {
  PS_TRY CHECK_KV(kv);
  if (ps_status rc = check_layer(kv, layer)) return rc;
  CallSeqs cs;
  if (ps_status rc = plan_seqs(kv, n_seqs, seqs, n_tok, -1, cs)) return rc;
  if (cs.rows > 0 && (!k || !v)) return fail(PS_E_INVALID, "null k or v");
  if (ps_status rc = check_aligned({k, v})) return rc;
  Meta mt;
  const size_t o_si = mt.add(cs.si.data(), cs.si.size() * sizeof(SeqInfo));
  const size_t o_bt = mt.add(cs.bt.data(), cs.bt.size() * 4);
  if (ps_status rc = check_ws(ws, ws_bytes, mt.size())) return rc;
  if (cs.rows == 0) return PS_OK;
  void* host;
  const int slot = kv->staging.acquire(mt.size(), &host);
  if (slot < 0) return PS_E_HIP;
  std::memcpy(host, mt.buf.data(), mt.buf.size());
  hipStream_t st = (hipStream_t)stream;
  if (ps_status rc = kv->staging.submit(slot, ws, mt.buf.size(), st)) return rc;
  char* w = (char*)ws;
  launch_kv_append(kv->cfg.dtype, cs.rows, k, v, kv->layer_base(layer), (const SeqInfo*)(w + o_si),
                   (const int32_t*)(w + o_bt), n_seqs, kv->cfg.n_kv_heads, kv->cfg.head_dim, st);
  return last_launch_error();
  PS_CATCH
}

extern "C" ps_status ps_kv_gather(ps_kv* kv, int32_t layer, int32_t seq, void* k_out, void* v_out, void* ws,
                                  size_t ws_bytes, void* stream) {
  PS_TRY CHECK_KV(kv);
  if (ps_status rc = check_layer(kv, layer)) return rc;
  std::string e;
  if (int rc = kv->meta.check_open(seq, e)) return fail(rc, e);
  const KvSeq& q = kv->meta.seq(seq);
  if (q.len > 0 && (!k_out || !v_out)) return fail(PS_E_INVALID, "null output");
  if (ps_status rc = check_aligned({k_out, v_out})) return rc;
  Meta mt;
  const int32_t pages = (q.len + 15) / 16;
  mt.add(q.pages.data(), pages * 4);
  if (ps_status rc = check_ws(ws, ws_bytes, mt.size())) return rc;
  if (q.len == 0) return PS_OK;
  void* host;
  const int slot = kv->staging.acquire(mt.size(), &host);
  if (slot < 0) return PS_E_HIP;
  std::memcpy(host, mt.buf.data(), mt.buf.size());
  hipStream_t st = (hipStream_t)stream;
  if (ps_status rc = kv->staging.submit(slot, ws, mt.buf.size(), st)) return rc;
  launch_kv_gather(kv->cfg.dtype, q.len, kv->layer_base(layer), (const int32_t*)ws, k_out, v_out,
                   kv->cfg.n_kv_heads, kv->cfg.head_dim, st);
  return last_launch_error();
  PS_CATCH
}

namespace {
ps_status upload_meta(ps_kv* kv, const Meta& mt, void* ws, hipStream_t st);
}  // namespace

extern "C" ps_status ps_kv_transfer(ps_kv* src, int32_t src_seq, ps_kv* dst, int32_t dst_seq, void* ws,
                                    size_t ws_bytes, void* stream) {
  PS_TRY
  if (!src || !dst) return fail(PS_E_INVALID, "null kv handle");
  if (!same_cfg(src->cfg, dst->cfg)) return fail(PS_E_INVALID, "source and destination pool configurations differ");
  if (src->n_layers != dst->n_layers) return fail(PS_E_INVALID, "source and destination pools differ in layer count");
  std::string e;
  if (int rc = src->meta.check_open(src_seq, e)) return fail(rc, "source: " + e);
  if (int rc = dst->meta.check_open(dst_seq, e)) return fail(rc, "destination: " + e);
  if (src == dst && src_seq == dst_seq) return fail(PS_E_INVALID, "source and destination are the same sequence");
  const int32_t len = src->meta.seq(src_seq).len;
  if (dst->meta.seq(dst_seq).len != 0) return fail(PS_E_INVALID, "destination sequence is not empty");
  if (int rc = dst->meta.check_writable(dst_seq, len, e)) return fail(rc, "destination: " + e);
  const int32_t pages = (len + PS_PAGE_TOKENS - 1) / PS_PAGE_TOKENS;
  Meta mt;
  const size_t o_sb = mt.add(src->meta.seq(src_seq).pages.data(), (size_t)pages * 4);
  const size_t o_db = mt.add(dst->meta.seq(dst_seq).pages.data(), (size_t)pages * 4);
  if (ps_status rc = check_ws(ws, ws_bytes, mt.size())) return rc;
  if (len > 0) {
    hipStream_t st = (hipStream_t)stream;
    if (ps_status rc = upload_meta(dst, mt, ws, st)) return rc;
    const ps_layer_cfg& c = src->cfg;
    const size_t eb = elt_bytes(c.dtype);
    const size_t page_bytes = (size_t)c.n_kv_heads * 2 * PS_PAGE_TOKENS * c.head_dim * eb;
    if (launch_kv_copy_pages(page_bytes, pages, src->n_layers, src->pool, src->layer_elts * eb,
                             (const int32_t*)((char*)ws + o_sb), dst->pool, dst->layer_elts * eb,
                             (const int32_t*)((char*)ws + o_db), st))
      return fail(PS_E_UNSUPPORTED, "page copy configuration not supported");
    if (ps_status rc = last_launch_error()) return rc;
  }
  // the copied positions become the destination's committed length
  if (int rc = dst->meta.commit(1, &dst_seq, &len, e)) return fail(rc, e);
  return PS_OK;
  PS_CATCH
}

// ------------------------------------------------------------ admission
struct ps_sched {
  ps_kv* kv;
  Admission adm;
  ps_sched(ps_kv* k, const ps_sched_cfg& c) : kv(k), adm(k->meta, c.window, c.cs_initial, c.cs_min, c.cs_max) {}
};

extern "C" ps_status ps_sched_create(ps_kv* kv, const ps_sched_cfg* c, ps_sched** out) {
  PS_TRY CHECK_KV(kv);
  if (!c || !out) return fail(PS_E_INVALID, "null argument");
  auto page_multiple = [](int32_t v) { return v > 0 && v % PS_PAGE_TOKENS == 0; };
  if (c->window < 1 || !page_multiple(c->cs_initial) || !page_multiple(c->cs_min) || !page_multiple(c->cs_max) ||
      c->cs_min > c->cs_max)
    return fail(PS_E_INVALID, "window >= 1 and positive chunk sizes in multiples of 16 with cs_min <= cs_max");
  *out = new ps_sched(kv, *c);
  return PS_OK;
  PS_CATCH
}
extern "C" ps_status ps_sched_destroy(ps_sched* s) {
  PS_TRY
  delete s;
  return PS_OK;
  PS_CATCH
}
#define CHECK_SCHED(s) \
  if (!(s)) return fail(PS_E_INVALID, "null scheduler handle");
extern "C" ps_status ps_sched_chunk_size(const ps_sched* s, int32_t* cs) {
  PS_TRY CHECK_SCHED(s);
  if (!cs) return fail(PS_E_INVALID, "null cs");
  *cs = s->adm.chunk_size();
  return PS_OK;
  PS_CATCH
}
extern "C" ps_status ps_sched_running(const ps_sched* s, int32_t* n) {
  PS_TRY CHECK_SCHED(s);
  if (!n) return fail(PS_E_INVALID, "null n");
  *n = s->adm.running();
  return PS_OK;
  PS_CATCH
}
extern "C" ps_status ps_sched_admit(ps_sched* s, int32_t ctx, int32_t* seq) {
  PS_TRY CHECK_SCHED(s);
  if (!seq) return fail(PS_E_INVALID, "null seq");
  std::string e;
  if (int rc = s->adm.admit(ctx, seq, e)) return fail(rc, e);
  return PS_OK;
  PS_CATCH
}
extern "C" ps_status ps_sched_reserve_step(ps_sched* s, int32_t n, const int32_t* seqs, const int32_t* n_tok,
                                           int32_t* preempted, int32_t cap, int32_t* n_preempted) {
  PS_TRY CHECK_SCHED(s);
  std::string e;
  if (int rc = s->adm.reserve_step(n, seqs, n_tok, cap, preempted, n_preempted, e)) return fail(rc, e);
  return PS_OK;
  PS_CATCH
}
extern "C" ps_status ps_sched_finish(ps_sched* s, int32_t seq, int32_t stage_tokens) {
  PS_TRY CHECK_SCHED(s);
  std::string e;
  if (int rc = s->adm.finish(seq, stage_tokens, e)) return fail(rc, e);
  return PS_OK;
  PS_CATCH
}

// ------------------------------------------------------ frequency control
struct ps_dvfs {
  Dvfs d;
  template <typename... A>
  explicit ps_dvfs(A&&... a) : d(std::forward<A>(a)...) {}
};

extern "C" ps_status ps_dvfs_create(const int32_t* ladder, int32_t n, double under_w, double over_w, int32_t limit_w,
                                    int32_t f0, ps_dvfs_lock_fn lock, ps_dvfs_limit_fn limit, void* ctx,
                                    ps_dvfs** out) {
  PS_TRY
  if (!ladder || n <= 0 || !out) return fail(PS_E_INVALID, "bad ladder or out");
  for (int i = 1; i < n; ++i)
    if (ladder[i] <= ladder[i - 1]) return fail(PS_E_INVALID, "ladder must increase strictly");
  if (!(under_w >= 0) || !(over_w >= 0)) return fail(PS_E_INVALID, "negative penalty weight");
  *out = new ps_dvfs(std::vector<int32_t>(ladder, ladder + n), under_w, over_w, limit_w, f0, lock, limit, ctx);
  return PS_OK;
  PS_CATCH
}
extern "C" ps_status ps_dvfs_destroy(ps_dvfs* d) {
  PS_TRY
  delete d;
  return PS_OK;
  PS_CATCH
}
#define CHECK_DVFS(d) \
  if (!(d)) return fail(PS_E_INVALID, "null dvfs handle");
extern "C" ps_status ps_dvfs_vote(ps_dvfs* d, int64_t r, int32_t target, double weight) {
  PS_TRY CHECK_DVFS(d);
  if (!(weight >= 0)) return fail(PS_E_INVALID, "negative vote weight");
  d->d.vote(r, target, weight);
  return PS_OK;
  PS_CATCH
}
extern "C" ps_status ps_dvfs_retract(ps_dvfs* d, int64_t r) {
  PS_TRY CHECK_DVFS(d);
  d->d.retract(r);
  return PS_OK;
  PS_CATCH
}
extern "C" ps_status ps_dvfs_tick(ps_dvfs* d, int32_t* mhz, int32_t* changed) {
  PS_TRY CHECK_DVFS(d);
  if (int32_t rc = d->d.tick(mhz, changed)) return fail(PS_E_HIP, "actuator returned " + std::to_string(rc));
  return PS_OK;
  PS_CATCH
}
extern "C" ps_status ps_dvfs_start(ps_dvfs* d, int32_t period_ms) {
  PS_TRY CHECK_DVFS(d);
  if (period_ms <= 0) return fail(PS_E_INVALID, "period must be positive");
  if (!d->d.start(period_ms)) return fail(PS_E_INVALID, "daemon already running");
  return PS_OK;
  PS_CATCH
}
extern "C" ps_status ps_dvfs_stop(ps_dvfs* d) {
  PS_TRY CHECK_DVFS(d);
  d->d.stop();
  return PS_OK;
  PS_CATCH
}

extern "C" ps_status ps_psopt_solve(const ps_psopt_group* g, int32_t n, double p_max, double f_min, double f_max,
                                    double dt, const int32_t* ladder, int32_t n_ladder, ps_psopt_result* out,
                                    double* mu, double* p_relaxed, double* p_projected) {
  PS_TRY
  if (!g || n <= 0 || !out || !ladder || n_ladder <= 0) return fail(PS_E_INVALID, "bad arguments");
  if (!(f_min > 0) || !(f_max > f_min) || !(p_max > 0) || !(dt >= 0)) return fail(PS_E_INVALID, "bad range");
  for (int i = 1; i < n_ladder; ++i)
    if (ladder[i] <= ladder[i - 1]) return fail(PS_E_INVALID, "ladder must increase strictly");
  for (int i = 0; i < n; ++i)
    if (!(g[i].k > 0) || !(g[i].c > 0) || !(g[i].gamma >= 0 && g[i].gamma <= 1) || !(g[i].lam > 0) ||
        !(g[i].sigma > 0) || !(g[i].delta >= 0) || !(g[i].w >= 0) || !(g[i].c2 >= 0) || !(g[i].c1 >= 0))
      return fail(PS_E_INVALID, "bad group " + std::to_string(i));
  if (int rc = psopt_solve(g, n, p_max, f_min, f_max, dt, ladder, n_ladder, out, mu, p_relaxed, p_projected))
    return fail(rc, "the power cap is not reachable at the frequencies the impact bounds allow");
  return PS_OK;
  PS_CATCH
}

// ------------------------------------------------------------------ layer
extern "C" ps_status ps_layer_create(const ps_layer_cfg* c, ps_layer** out) {
  PS_TRY
  if (ps_status rc = check_cfg(c)) return rc;
  if (!out) return fail(PS_E_INVALID, "null out");
  ps_layer* L = new ps_layer;
  L->cfg = *c;
  *out = L;
  return PS_OK;
  PS_CATCH
}

extern "C" ps_status ps_layer_destroy(ps_layer* L) {
  PS_TRY
  delete L;
  return PS_OK;
  PS_CATCH
}

extern "C" size_t ps_workspace_bytes(const ps_layer_cfg* c, int32_t max_rows, int32_t max_seqs,
                                     int32_t max_pages_per_seq) {
  if (!c || max_rows < 0 || max_seqs < 0 || max_pages_per_seq < 0) return 0;
  const size_t mb = meta_bound(*c, max_rows, max_seqs, max_pages_per_seq);
  const int32_t parts = max_seqs * ((max_pages_per_seq + 7) / 8);
  return layout(*c, mb, max_rows, parts).total;
}

namespace {

// Everything a layer call needs besides weights, pool and activations: the
// call's sequence tables and work lists (uploaded once to the workspace head)
// and the workspace carve-out. A model step plans once and launches it for
// every layer.
struct LayerPlan {
  int32_t rows = 0, chunk_rows = 0, n_chunk = 0, n_dec = 0;
  bool fa = false, dec_mfma = false;
  size_t o_si = 0, o_bt = 0, o_fr = 0, o_pi = 0, o_di = 0, o_pb = 0, o_pc = 0;
  int n_pitems = 0, n_ditems = 0;
  int32_t n_parts = 0;
  int32_t n_seqs = 0;
  Meta mt;
  WsLayout wl;
};

ps_status plan_layer(const ps_layer_cfg& c, const ps_kv* kv, int32_t phase, int32_t n_chunk,
                     const int32_t* chunk_seqs, const int32_t* chunk_tok, int32_t n_dec, const int32_t* dec_seqs,
                     LayerPlan& P) {
  if (phase < PS_PHASE_PREFILL || phase > PS_PHASE_ANSWER) return fail(PS_E_INVALID, "bad phase");
  CallSeqs cs;
  if (ps_status rc = plan_seqs(kv, n_chunk, chunk_seqs, chunk_tok, -1, cs)) return rc;
  P.chunk_rows = cs.rows;
  if (ps_status rc = plan_seqs(kv, n_dec, dec_seqs, nullptr, 1, cs)) return rc;
  for (int i = 0; i < n_dec; ++i)
    for (int j = 0; j < n_chunk; ++j)
      if (dec_seqs[i] == chunk_seqs[j]) return fail(PS_E_INVALID, "sequence both chunked and decoding");
  P.rows = cs.rows;
  P.n_chunk = n_chunk;
  P.n_dec = n_dec;
  P.n_seqs = (int32_t)cs.si.size();
  const int d = c.hidden, dq = c.n_q_heads * c.head_dim, dkv = c.n_kv_heads * c.head_dim;
  // every GEMM of the call must be supported before anything is enqueued
  if (P.rows > 0 && (gemm_check(c.dtype, 0, P.rows, dq + 2 * dkv, d) || gemm_check(c.dtype, 1, P.rows, d, dq) ||
                     gemm_check(c.dtype, 2, P.rows, 2 * c.ffn, d) || gemm_check(c.dtype, 1, P.rows, d, c.ffn)))
    return fail(PS_E_UNSUPPORTED, "GEMM shape not supported by libps");
  P.o_si = P.mt.add(cs.si.data(), cs.si.size() * sizeof(SeqInfo));
  P.o_bt = P.mt.add(cs.bt.data(), cs.bt.size() * 4);
  const std::vector<double> fr = inv_freq(c);
  P.o_fr = P.mt.add(fr.data(), fr.size() * 8);
  P.fa = fa_ok(c) && n_chunk > 0;
  P.dec_mfma = dec_ok(c) && n_dec > 0;
  if (P.fa) {
    std::vector<PrefillItem> pitems = plan_prefill(cs.si, n_chunk);
    P.n_pitems = (int)pitems.size();
    P.o_pi = P.mt.add(pitems.data(), pitems.size() * sizeof(PrefillItem));
  }
  if (P.dec_mfma) {
    DecodePlan dp = plan_decode(cs.si, n_chunk, choose_split_pages(cs.si, n_chunk, c.n_kv_heads, phase));
    if ((long)dp.items.size() > kMaxDecodeItems)
      return fail(PS_E_UNSUPPORTED, "decode batch exceeds 65535 attention work items");
    P.n_ditems = (int)dp.items.size();
    P.n_parts = dp.n_parts;
    P.o_di = P.mt.add(dp.items.data(), dp.items.size() * sizeof(DecodeItem));
    P.o_pb = P.mt.add(dp.part_begin.data(), dp.part_begin.size() * 4);
    P.o_pc = P.mt.add(dp.part_count.data(), dp.part_count.size() * 4);
  }
  return PS_OK;
}

ps_status upload_meta(ps_kv* kv, const Meta& mt, void* ws, hipStream_t st) {
  void* host;
  const int slot = kv->staging.acquire(mt.size(), &host);
  if (slot < 0) return PS_E_HIP;
  std::memcpy(host, mt.buf.data(), mt.buf.size());
  return kv->staging.submit(slot, ws, mt.buf.size(), st);
}

// upload_meta, except that the upload is returned as a job for the caller's
// first kernel to carry (which must then be enqueued).
ps_status stage_meta(ps_kv* kv, const Meta& mt, void* ws, UploadJob* job) {
  void* host;
  const int slot = kv->staging.acquire(mt.size(), &host);
  if (slot < 0) return PS_E_HIP;
  std::memcpy(host, mt.buf.data(), mt.buf.size());
  return kv->staging.prepare(slot, ws, mt.buf.size(), job);
}

// The kernels of one layer: x_in -> x_out for the planned rows.
// `up`, if given, is the call's metadata upload: the first kernel carries it
// (every kernel that reads the metadata runs after that one).
int launch_layer(const ps_layer_cfg& c, const LayerPlan& P, const ps_layer_w* w, void* pool, const void* x_in,
                 void* x_out, char* W, hipStream_t st, const UploadJob* up = nullptr, AuxStream* aux = nullptr) {
  const WsLayout& wl = P.wl;
  const int d = c.hidden, dq = c.n_q_heads * c.head_dim, dkv = c.n_kv_heads * c.head_dim;
  const int dt = c.dtype, G = group_of(c), rows = P.rows;
  const SeqInfo* si = (const SeqInfo*)(W + P.o_si);
  const int32_t* bt = (const int32_t*)(W + P.o_bt);
  char* xn = W + wl.xn;
  void* qkv = W + wl.qkv;
  char* qr = W + wl.qr;
  char* o = W + wl.o;
  char* h = W + wl.h;
  char* m = W + wl.m;
  void* gws = W + wl.gemm;
  const size_t gws_bytes = wl.gemm_b - wl.gemm;
  void* gws_b = W + wl.gemm_b;
  const size_t gws_b_bytes = wl.apart_o - wl.gemm_b;
  const size_t eb = elt_bytes(dt);
  const float scale = 1.0f / std::sqrt((float)c.head_dim);
  const float scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)c.head_dim));
  // bf16, d a multiple of 8 up to 8192: a row fits the fused split-sum +
  // residual + RMSNorm kernel's registers
  const bool fused_norm = dt == PS_BF16 && d % 8 == 0 && d <= 8192;
  int bad = 0;

  // O projection + residual -> h (fp32), then the FFN RMSNorm -> xn, over
  // `n` rows from row r0. Split-K partials (a decode-sized skinny plan, or a
  // tile launch that would leave compute units idle) are summed by the norm
  // kernel, which also adds the residual and stores h.
  auto o_proj = [&](int r0, int n, void* ws, size_t ws_bytes, hipStream_t s) {
    if (n == 0) return;
    const char* a = o + (size_t)r0 * dq * eb;
    const char* res = (const char*)x_in + (size_t)r0 * d * eb;
    float* hr = (float*)(h + (size_t)r0 * d * 4);
    char* y = xn + (size_t)r0 * d * eb;
    int S = 1;
    if (fused_norm) {
      S = gemm_tile_splits(n, d, dq);
      if (S > 1) {
        if (ws_bytes < (size_t)S * n * d * 4) {  // the layout's bound rules this out
          bad |= 1;
          return;
        }
        bad |= launch_gemm_tile_split(n, d, dq, S, a, w->w_o, (float*)ws, s);
      } else {
        bad |= launch_gemm_split(dt, dt, PS_F32, PS_EPI_RESIDUAL, n, d, dq, a, w->w_o, res, hr, ws, ws_bytes, s, &S);
      }
    } else {
      bad |= launch_gemm(dt, dt, PS_F32, PS_EPI_RESIDUAL, n, d, dq, a, w->w_o, res, hr, ws, ws_bytes, s);
    }
    if (S > 1)
      bad |= launch_split_residual_rmsnorm(n, d, S, (const float*)ws, res, hr, w->ffn_norm, c.rms_eps, y, s);
    else
      bad |= launch_rmsnorm(PS_F32, dt, dt, n, d, hr, w->ffn_norm, c.rms_eps, y, s);
  };
  // down projection + residual (h) -> x_out over `n` rows from row r0
  auto down_proj = [&](int r0, int n, void* ws, size_t ws_bytes, hipStream_t s) {
    if (n == 0) return;
    const char* a = m + (size_t)r0 * c.ffn * eb;
    const float* hr = (const float*)(h + (size_t)r0 * d * 4);
    char* y = (char*)x_out + (size_t)r0 * d * eb;
    const int S = dt == PS_BF16 ? gemm_tile_splits(n, d, c.ffn) : 1;
    if (S > 1) {
      if (ws_bytes < (size_t)S * n * d * 4) {  // the layout's bound rules this out
        bad |= 1;
        return;
      }
      bad |= launch_gemm_tile_split(n, d, c.ffn, S, a, w->w_down, (float*)ws, s);
      bad |= launch_split_residual(PS_F32, dt, n, d, S, (const float*)ws, hr, y, s);
    } else {
      bad |= launch_gemm(dt, PS_F32, dt, PS_EPI_RESIDUAL, n, d, c.ffn, a, w->w_down, hr, y, ws, ws_bytes, s);
    }
  };
  auto prefill_attn = [&](hipStream_t s) {
    if (P.fa)
      bad |= launch_fa_prefill(G, P.n_pitems, c.n_kv_heads, qr, pool, si, bt, (const PrefillItem*)(W + P.o_pi), o,
                               scale_log2, s);
    else
      bad |= launch_attn_generic(dt, 0, P.chunk_rows, P.n_seqs, c.n_q_heads, c.n_kv_heads, c.head_dim, qr, pool, si,
                                 bt, o, scale, s);
  };
  auto decode_attn = [&](hipStream_t s, int max_wg) {
    if (P.dec_mfma) {
      const char* qd = qr + (size_t)P.chunk_rows * dq * eb;
      char* od = o + (size_t)P.chunk_rows * dq * eb;
      bad |= launch_decode_attn(G, P.n_ditems, c.n_kv_heads, P.n_dec, qd, pool, si + P.n_chunk, bt,
                                (const DecodeItem*)(W + P.o_di), (float*)(W + wl.apart_o), (float*)(W + wl.apart_ml),
                                (const int32_t*)(W + P.o_pb), (const int32_t*)(W + P.o_pc), od, scale_log2, s,
                                max_wg);
    } else {
      bad |= launch_attn_generic(dt, P.chunk_rows, P.n_dec, P.n_seqs, c.n_q_heads, c.n_kv_heads, c.head_dim, qr,
                                 pool, si, bt, o, scale, s);
    }
  };

  bad |= launch_rmsnorm(dt, dt, dt, rows, d, x_in, w->attn_norm, c.rms_eps, xn, st, up);
  // decode-sized QKV: RoPE + KV write sums the split-K partials itself
  // (bf16, head_dim a multiple of 8: the fused reader's vector width)
  int s_qkv = 1;
  if (dt == PS_BF16 && c.head_dim % 8 == 0)
    bad |= launch_gemm_split(dt, 0, dt, PS_EPI_STORE, rows, dq + 2 * dkv, d, xn, w->w_qkv, nullptr, qkv, gws,
                             gws_bytes, st, &s_qkv);
  else
    bad |= launch_gemm(dt, 0, dt, PS_EPI_STORE, rows, dq + 2 * dkv, d, xn, w->w_qkv, nullptr, qkv, gws, gws_bytes, st);
  bad |= launch_rope_kvwrite(dt, rows, qkv, qr, pool, si, bt, (const double*)(W + P.o_fr), P.n_seqs, c.n_q_heads,
                             c.n_kv_heads, c.head_dim, st, (const float*)gws, s_qkv);

  // A mixed batch (prefill chunks + decode rows) splits after the KV write:
  // the decode rows' attention (HBM-bound over long contexts) and the rest
  // of their layer (skinny O, SwiGLU and down GEMMs, weight-bandwidth
  // bound) run on the second stream while the chunk rows' flash attention
  // and tile GEMMs run on the caller's. The two row sets write disjoint rows
  // of o, h, xn, m and x_out, and each stream has its own split-K partials.
  const bool fork = aux && P.n_chunk > 0 && P.n_dec > 0 && P.n_dec <= 64 && P.chunk_rows > 64 && fused_norm;
  if (!fork) {
    if (P.n_chunk > 0) prefill_attn(st);
    if (P.n_dec > 0) decode_attn(st, 0);
    o_proj(0, rows, gws, gws_bytes, st);
    bad |= launch_gemm(dt, 0, dt, PS_EPI_SWIGLU, rows, 2 * c.ffn, d, xn, w->w_gate_up, nullptr, m, gws, gws_bytes,
                       st);
    down_proj(0, rows, gws, gws_bytes, st);
    return bad;
  }
  const hipStream_t sb = aux->s;
  const int cr = P.chunk_rows;
  auto link = [&](hipStream_t from, hipStream_t to, int i) {  // `to` waits for the work enqueued on `from` so far
    if (hipEventRecord(aux->ev[i], from) != hipSuccess || hipStreamWaitEvent(to, aux->ev[i], 0) != hipSuccess)
      bad |= 1;
  };
  auto swiglu = [&](int r0, int n, void* ws, size_t ws_bytes, hipStream_t s) {
    bad |= launch_gemm(dt, 0, dt, PS_EPI_SWIGLU, n, 2 * c.ffn, d, xn + (size_t)r0 * d * eb, w->w_gate_up, nullptr,
                       m + (size_t)r0 * c.ffn * eb, ws, ws_bytes, s);
  };
  link(st, sb, 0);
  // the decode rows' attention on at most half as many workgroups as compute
  // units, each walking several split items, so that it leaves compute units
  // to the chunk rows' GEMMs (uncapped it takes them all while it runs)
  decode_attn(sb, compute_units() / 2);
  o_proj(cr, P.n_dec, gws_b, gws_b_bytes, sb);
  swiglu(cr, P.n_dec, gws_b, gws_b_bytes, sb);
  down_proj(cr, P.n_dec, gws_b, gws_b_bytes, sb);
  prefill_attn(st);
  o_proj(0, cr, gws, gws_bytes, st);
  swiglu(0, cr, gws, gws_bytes, st);
  down_proj(0, cr, gws, gws_bytes, st);
  link(sb, st, 1);  // joined: the call's work is on the caller's stream again
  return bad;
}

ps_status check_weights(const ps_layer_w* w) {
  if (!w || !w->attn_norm || !w->w_qkv || !w->w_o || !w->ffn_norm || !w->w_gate_up || !w->w_down)
    return fail(PS_E_INVALID, "null weight pointer");
  return check_aligned({w->attn_norm, w->w_qkv, w->w_o, w->ffn_norm, w->w_gate_up, w->w_down});
}

// One layer over n_chunk prefill sequences (chunk_tok rows each) followed by
// n_dec decode sequences (one row each).
ps_status run_layer(ps_layer* L, const ps_layer_w* w, ps_kv* kv, int32_t layer, int32_t phase, int32_t n_chunk,
                    const int32_t* chunk_seqs, const int32_t* chunk_tok, int32_t n_dec, const int32_t* dec_seqs,
                    const void* x_in, void* x_out, void* ws, size_t ws_bytes, void* stream) {
  if (!L) return fail(PS_E_INVALID, "null layer handle");
  CHECK_KV(kv);
  if (ps_status rc = check_weights(w)) return rc;
  const ps_layer_cfg& c = L->cfg;
  if (!same_cfg(c, kv->cfg))
    return fail(PS_E_INVALID, "layer and KV pool configurations differ");
  if (ps_status rc = check_layer(kv, layer)) return rc;
  LayerPlan P;
  if (ps_status rc = plan_layer(c, kv, phase, n_chunk, chunk_seqs, chunk_tok, n_dec, dec_seqs, P)) return rc;
  if (P.rows == 0) return PS_OK;
  if (!x_in || !x_out) return fail(PS_E_INVALID, "null activation pointer");
  if (ps_status rc = check_aligned({x_in, x_out})) return rc;
  P.wl = layout(c, P.mt.size(), P.rows, P.n_parts);
  if (ps_status rc = check_ws(ws, ws_bytes, P.wl.total)) return rc;
  hipStream_t st = (hipStream_t)stream;
  AuxStream* aux = nullptr;
  if (n_chunk > 0 && n_dec > 0)
    if (ps_status rc = L->aux.get(st, &aux)) return rc;
  UploadJob up;
  if (ps_status rc = stage_meta(kv, P.mt, ws, &up)) return rc;
  if (launch_layer(c, P, w, kv->layer_base(layer), x_in, x_out, (char*)ws, st, &up, aux))
    return fail(PS_E_UNSUPPORTED, "a kernel rejected its configuration");
  return last_launch_error();
}

}  // namespace

// ------------------------------------------------------------------ model
namespace {

struct ModelWs {
  size_t xa, xb, hl, hn, logits, lm, total;
};

ModelWs model_layout(const ps_layer_cfg& c, int32_t vocab, size_t layer_total, int32_t rows, int32_t n_out) {
  ModelWs m;
  size_t off = align_up(layer_total, 256);
  auto take = [&](size_t bytes) {
    size_t o = off;
    off = align_up(off + bytes, 256);
    return o;
  };
  m.xa = take((size_t)rows * c.hidden * 2);
  m.xb = take((size_t)rows * c.hidden * 2);
  m.hl = take((size_t)n_out * c.hidden * 2);
  m.hn = take((size_t)n_out * c.hidden * 2);
  m.logits = take((size_t)n_out * vocab * 4);
  m.lm = take(gemm_workspace_bytes(PS_BF16, n_out, vocab, c.hidden));
  m.total = off;
  return m;
}

ps_status run_model(ps_model* M, ps_kv* kv, int32_t phase, int32_t n_chunk, const int32_t* chunk_seqs,
                    const int32_t* chunk_tok, int32_t n_dec, const int32_t* dec_seqs, const int32_t* tokens,
                    int32_t* next, float* logits_out, void* ws, size_t ws_bytes, void* stream) {
  if (!M) return fail(PS_E_INVALID, "null model handle");
  CHECK_KV(kv);
  const ps_layer_cfg& c = M->cfg;
  if (!same_cfg(c, kv->cfg)) return fail(PS_E_INVALID, "model and KV pool configurations differ");
  if (kv->n_layers < M->n_layers) return fail(PS_E_INVALID, "KV pool has fewer layers than the model");
  LayerPlan P;
  if (ps_status rc = plan_layer(c, kv, phase, n_chunk, chunk_seqs, chunk_tok, n_dec, dec_seqs, P)) return rc;
  if (P.rows == 0) return PS_OK;
  if (!tokens || !next) return fail(PS_E_INVALID, "null token pointer");
  if (ps_status rc = check_aligned({logits_out})) return rc;
  const int32_t n_out = n_chunk + n_dec;
  if (gemm_check(PS_BF16, PS_EPI_STORE, n_out, M->vocab, c.hidden))
    return fail(PS_E_UNSUPPORTED, "LM head shape not supported by libps");
  // last row of every sequence feeds the LM head
  std::vector<int32_t> last(n_out);
  {
    int32_t r = 0;
    for (int i = 0; i < n_chunk; ++i) {
      r += chunk_tok[i];
      last[i] = r - 1;
    }
    for (int i = 0; i < n_dec; ++i) last[n_chunk + i] = r + i;
  }
  const size_t o_last = P.mt.add(last.data(), last.size() * 4);
  P.wl = layout(c, P.mt.size(), P.rows, P.n_parts);
  const ModelWs mw = model_layout(c, M->vocab, P.wl.total, P.rows, n_out);
  if (ps_status rc = check_ws(ws, ws_bytes, mw.total)) return rc;
  hipStream_t st = (hipStream_t)stream;
  if (ps_status rc = upload_meta(kv, P.mt, ws, st)) return rc;
  char* W = (char*)ws;
  int bad = launch_embed(P.rows, c.hidden, M->vocab, M->embed, tokens, W + mw.xa, st);
  char* cur = W + mw.xa;
  char* nxt = W + mw.xb;
  for (int l = 0; l < M->n_layers; ++l) {
    bad |= launch_layer(c, P, &M->layers[l], kv->layer_base(l), cur, nxt, W, st);
    std::swap(cur, nxt);
  }
  float* logits = logits_out ? logits_out : (float*)(W + mw.logits);
  bad |= launch_gather_rows(n_out, c.hidden, cur, (const int32_t*)(W + o_last), W + mw.hl, st);
  bad |= launch_rmsnorm(PS_BF16, PS_BF16, PS_BF16, n_out, c.hidden, W + mw.hl, M->final_norm, c.rms_eps, W + mw.hn,
                        st);
  bad |= launch_gemm(PS_BF16, 0, PS_F32, PS_EPI_STORE, n_out, M->vocab, c.hidden, W + mw.hn, M->lm_head, nullptr,
                     logits, W + mw.lm, mw.total - mw.lm, st);
  bad |= launch_argmax(n_out, M->vocab, logits, next, st);
  if (bad) return fail(PS_E_UNSUPPORTED, "a kernel rejected its configuration");
  return last_launch_error();
}

}  // namespace

extern "C" ps_status ps_model_create(const ps_layer_cfg* c, int32_t n_layers, int32_t vocab, const void* embed,
                                     const ps_layer_w* layers, const void* final_norm, const void* lm_head,
                                     ps_model** out) {
  PS_TRY
  if (ps_status rc = check_cfg(c)) return rc;
  if (c->dtype != PS_BF16) return fail(PS_E_UNSUPPORTED, "the model path is bf16");
  if (c->hidden % 8) return fail(PS_E_UNSUPPORTED, "hidden must be a multiple of 8");
  if (!out || n_layers <= 0 || vocab <= 0 || !embed || !layers || !final_norm || !lm_head)
    return fail(PS_E_INVALID, "bad model arguments");
  for (int l = 0; l < n_layers; ++l)
    if (ps_status rc = check_weights(&layers[l])) return rc;
  if (ps_status rc = check_aligned({embed, final_norm, lm_head})) return rc;
  ps_model* M = new ps_model;
  M->cfg = *c;
  M->n_layers = n_layers;
  M->vocab = vocab;
  M->embed = embed;
  M->final_norm = final_norm;
  M->lm_head = lm_head;
  M->layers.assign(layers, layers + n_layers);
  *out = M;
  return PS_OK;
  PS_CATCH
}

extern "C" ps_status ps_model_destroy(ps_model* M) {
  PS_TRY
  delete M;
  return PS_OK;
  PS_CATCH
}

extern "C" size_t ps_model_workspace_bytes(const ps_layer_cfg* c, int32_t vocab, int32_t max_rows, int32_t max_seqs,
                                           int32_t max_pages_per_seq) {
  if (!c || vocab <= 0 || max_rows < 0 || max_seqs < 0 || max_pages_per_seq < 0) return 0;
  const size_t mb = meta_bound(*c, max_rows, max_seqs, max_pages_per_seq) + align_up(4ull * max_seqs, 256);
  const int32_t parts = max_seqs * ((max_pages_per_seq + 7) / 8);
  const WsLayout wl = layout(*c, mb, max_rows, parts);
  return model_layout(*c, vocab, wl.total, max_rows, max_seqs).total;
}

extern "C" ps_status ps_model_prefill(ps_model* M, ps_kv* kv, int32_t n_seqs, const int32_t* seqs,
                                      const int32_t* n_tok, const int32_t* dev_tokens, int32_t* dev_next,
                                      float* dev_logits, void* ws, size_t ws_bytes, void* stream) {
  PS_TRY
  return run_model(M, kv, PS_PHASE_PREFILL, n_seqs, seqs, n_tok, 0, nullptr, dev_tokens, dev_next, dev_logits, ws,
                   ws_bytes, stream);
  PS_CATCH
}

extern "C" ps_status ps_model_decode_step(ps_model* M, ps_kv* kv, int32_t phase, int32_t n_seqs, const int32_t* seqs,
                                          const int32_t* dev_tokens, int32_t* dev_next, float* dev_logits, void* ws,
                                          size_t ws_bytes, void* stream) {
  PS_TRY
  return run_model(M, kv, phase, 0, nullptr, nullptr, n_seqs, seqs, dev_tokens, dev_next, dev_logits, ws, ws_bytes,
                   stream);
  PS_CATCH
}

extern "C" ps_status ps_op_argmax(int32_t rows, int32_t vocab, const float* logits, int32_t* next, void* stream) {
  PS_TRY
  if (rows < 0 || vocab <= 0) return fail(PS_E_INVALID, "bad shape");
  if (rows > 0 && (!logits || !next)) return fail(PS_E_INVALID, "null pointer");
  launch_argmax(rows, vocab, logits, next, (hipStream_t)stream);
  return last_launch_error();
  PS_CATCH
}

extern "C" ps_status ps_prefill(ps_layer* L, const ps_layer_w* w, ps_kv* kv, int32_t layer, int32_t n_seqs,
                                const int32_t* seqs, const int32_t* n_tok, const void* x_in, void* x_out, void* ws,
                                size_t ws_bytes, void* stream) {
  PS_TRY
  return run_layer(L, w, kv, layer, PS_PHASE_PREFILL, n_seqs, seqs, n_tok, 0, nullptr, x_in, x_out, ws, ws_bytes,
                   stream);
  PS_CATCH
}

extern "C" ps_status ps_decode_step(ps_layer* L, const ps_layer_w* w, ps_kv* kv, int32_t layer, int32_t phase,
                                    int32_t n_seqs, const int32_t* seqs, const void* x_in, void* x_out, void* ws,
                                    size_t ws_bytes, void* stream) {
  PS_TRY
  return run_layer(L, w, kv, layer, phase, 0, nullptr, nullptr, n_seqs, seqs, x_in, x_out, ws, ws_bytes, stream);
  PS_CATCH
}

extern "C" ps_status ps_mixed_step(ps_layer* L, const ps_layer_w* w, ps_kv* kv, int32_t layer, int32_t n_chunk,
                                   const int32_t* chunk_seqs, const int32_t* chunk_tok, int32_t n_dec,
                                   const int32_t* dec_seqs, const void* x_in, void* x_out, void* ws,
                                   size_t ws_bytes, void* stream) {
  PS_TRY
  return run_layer(L, w, kv, layer, PS_PHASE_THINK, n_chunk, chunk_seqs, chunk_tok, n_dec, dec_seqs, x_in, x_out,
                   ws, ws_bytes, stream);
  PS_CATCH
}

// ------------------------------------------------------------------ ops
extern "C" ps_status ps_op_rmsnorm(int32_t x_dt, int32_t g_dt, int32_t y_dt, int32_t rows, int32_t d,
                                   const void* x, const void* g, float eps, void* y, void* stream) {
  PS_TRY
  if (rows < 0 || d <= 0) return fail(PS_E_INVALID, "bad shape");
  if (rows > 0 && (!x || !g || !y)) return fail(PS_E_INVALID, "null pointer");
  if (ps_status rc = check_aligned({x, g, y})) return rc;
  for (int dt : {x_dt, g_dt, y_dt})
    if (dt != PS_F32 && dt != PS_BF16) return fail(PS_E_INVALID, "bad dtype");
  if (launch_rmsnorm(x_dt, g_dt, y_dt, rows, d, x, g, eps, y, (hipStream_t)stream))
    return fail(PS_E_UNSUPPORTED, "dtype combination not supported");
  return last_launch_error();
  PS_CATCH
}

extern "C" size_t ps_op_gemm_workspace_bytes(int32_t dtype, int32_t M, int32_t N, int32_t K) {
  if (M < 0 || N <= 0 || K <= 0) return 0;
  return gemm_workspace_bytes(dtype, M, N, K);
}

extern "C" ps_status ps_op_gemm(int32_t dtype, int32_t r_dt, int32_t c_dt, int32_t epi, int32_t M, int32_t N,
                                int32_t K, const void* A, const void* Wt, const void* R, void* C, void* ws,
                                size_t ws_bytes, void* stream) {
  PS_TRY
  if (epi < 0 || epi > 2) return fail(PS_E_INVALID, "bad epilogue");
  if (M > 0 && (!A || !Wt || !C || (epi == 1 && !R))) return fail(PS_E_INVALID, "null pointer");
  if (ps_status rc = check_aligned({A, Wt, R, C, ws})) return rc;
  if (gemm_check(dtype, epi, M, N, K)) return fail(PS_E_UNSUPPORTED, "GEMM shape not supported");
  const size_t need = gemm_workspace_bytes(dtype, M, N, K);
  if (need && (!ws || ws_bytes < need)) return fail(PS_E_INVALID, "workspace too small for split-K partials");
  if (epi != 1) r_dt = 0;
  int rc = launch_gemm(dtype, r_dt, c_dt, epi, M, N, K, A, Wt, R, C, ws, ws_bytes, (hipStream_t)stream);
  if (rc) return fail(PS_E_UNSUPPORTED, "dtype/epilogue combination not supported");
  return last_launch_error();
  PS_CATCH
}

static_assert(kGemmStaticScratchBytes == PS_GEMM_STATIC_SCRATCH_BYTES, "static scratch size");

extern "C" ps_status ps_op_gemm_static(int32_t dtype, int32_t r_dt, int32_t c_dt, int32_t epi, int32_t M, int32_t N,
                                       int32_t K, const void* A, const void* Wt, const void* R, void* C,
                                       void* stream) {
  PS_TRY
  if (epi < 0 || epi > 2) return fail(PS_E_INVALID, "bad epilogue");
  if (M > 0 && (!A || !Wt || !C || (epi == 1 && !R))) return fail(PS_E_INVALID, "null pointer");
  if (ps_status rc = check_aligned({A, Wt, R, C})) return rc;
  if (gemm_check(dtype, epi, M, N, K)) return fail(PS_E_UNSUPPORTED, "GEMM shape not supported");
  const size_t need = gemm_partials_bytes(dtype, epi, M, N, K);
  if (need > PS_GEMM_STATIC_SCRATCH_BYTES)
    return fail(PS_E_INVALID, "split-K partials need " + std::to_string(need) +
                                  " bytes, more than the static scratch holds (PS_GEMM_STATIC_SCRATCH_BYTES); "
                                  "use ps_op_gemm with a workspace");
  if (M == 0) return PS_OK;
  hipStream_t st = (hipStream_t)stream;
  void* scratch = nullptr;
  if (need) {
    // the scratch copy is per device: the stream must run on the current one
    if (st) {
      int cur = 0, sdev = 0;
      hipError_t e = hipGetDevice(&cur);
      if (e == hipSuccess) e = hipStreamGetDevice(st, &sdev);
      if (e != hipSuccess) return hip_fail(e, "stream device");
      if (sdev != cur) return fail(PS_E_INVALID, "the stream belongs to another device than the current one");
    }
    if (hipError_t e = gemm_static_scratch(&scratch)) return hip_fail(e, "static scratch address");
  }
  if (epi != 1) r_dt = 0;
  int rc = launch_gemm(dtype, r_dt, c_dt, epi, M, N, K, A, Wt, R, C, scratch, need, st);
  if (rc) return fail(PS_E_UNSUPPORTED, "dtype/epilogue combination not supported");
  return last_launch_error();
  PS_CATCH
}

extern "C" ps_status ps_op_tile_weight(int32_t dtype, int32_t N, int32_t K, const void* w, void* out, void* stream) {
  PS_TRY
  if (!w || !out || N <= 0 || K <= 0 || (dtype != PS_F32 && dtype != PS_BF16))
    return fail(PS_E_INVALID, "bad arguments");
  if (ps_status rc = check_aligned({w, out})) return rc;
  if (launch_tile_weight(elt_bytes(dtype), N, K, w, out, (hipStream_t)stream))
    return fail(PS_E_UNSUPPORTED, "element size");
  return last_launch_error();
  PS_CATCH
}

extern "C" ps_status ps_op_rope_kvwrite(ps_kv* kv, int32_t layer, int32_t n_seqs, const int32_t* seqs,
                                        const int32_t* n_tok, const void* qkv, void* q_out, void* ws,
                                        size_t ws_bytes, void* stream) {
  PS_TRY CHECK_KV(kv);
  if (ps_status rc = check_layer(kv, layer)) return rc;
  CallSeqs cs;
  if (ps_status rc = plan_seqs(kv, n_seqs, seqs, n_tok, -1, cs)) return rc;
  if (cs.rows > 0 && (!qkv || !q_out)) return fail(PS_E_INVALID, "null pointer");
  if (ps_status rc = check_aligned({qkv, q_out})) return rc;
  Meta mt;
  const size_t o_si = mt.add(cs.si.data(), cs.si.size() * sizeof(SeqInfo));
  const size_t o_bt = mt.add(cs.bt.data(), cs.bt.size() * 4);
  const std::vector<double> fr = inv_freq(kv->cfg);
  const size_t o_fr = mt.add(fr.data(), fr.size() * 8);
  if (ps_status rc = check_ws(ws, ws_bytes, mt.size())) return rc;
  if (cs.rows == 0) return PS_OK;
  void* host;
  const int slot = kv->staging.acquire(mt.size(), &host);
  if (slot < 0) return PS_E_HIP;
  std::memcpy(host, mt.buf.data(), mt.buf.size());
  hipStream_t st = (hipStream_t)stream;
  if (ps_status rc = kv->staging.submit(slot, ws, mt.buf.size(), st)) return rc;
  char* W = (char*)ws;
  const ps_layer_cfg& c = kv->cfg;
  launch_rope_kvwrite(c.dtype, cs.rows, qkv, q_out, kv->layer_base(layer), (const SeqInfo*)(W + o_si),
                      (const int32_t*)(W + o_bt), (const double*)(W + o_fr), n_seqs, c.n_q_heads, c.n_kv_heads,
                      c.head_dim, st);
  return last_launch_error();
  PS_CATCH
}

extern "C" ps_status ps_op_attention(ps_kv* kv, int32_t layer, int32_t n_seqs, const int32_t* seqs,
                                     const int32_t* n_tok, const void* q, void* o, void* ws, size_t ws_bytes,
                                     void* stream) {
  PS_TRY CHECK_KV(kv);
  if (ps_status rc = check_layer(kv, layer)) return rc;
  CallSeqs cs;
  if (ps_status rc = plan_seqs(kv, n_seqs, seqs, n_tok, -1, cs)) return rc;
  if (cs.rows > 0 && (!q || !o)) return fail(PS_E_INVALID, "null pointer");
  if (ps_status rc = check_aligned({q, o})) return rc;
  const ps_layer_cfg& c = kv->cfg;
  Meta mt;
  const size_t o_si = mt.add(cs.si.data(), cs.si.size() * sizeof(SeqInfo));
  const size_t o_bt = mt.add(cs.bt.data(), cs.bt.size() * 4);
  const bool fa = fa_ok(c);
  std::vector<PrefillItem> pitems;
  size_t o_pi = 0;
  if (fa) {
    pitems = plan_prefill(cs.si, cs.si.size());
    o_pi = mt.add(pitems.data(), pitems.size() * sizeof(PrefillItem));
  }
  if (ps_status rc = check_ws(ws, ws_bytes, mt.size())) return rc;
  if (cs.rows == 0) return PS_OK;
  void* host;
  const int slot = kv->staging.acquire(mt.size(), &host);
  if (slot < 0) return PS_E_HIP;
  std::memcpy(host, mt.buf.data(), mt.buf.size());
  hipStream_t st = (hipStream_t)stream;
  if (ps_status rc = kv->staging.submit(slot, ws, mt.buf.size(), st)) return rc;
  char* W = (char*)ws;
  const float scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)c.head_dim));
  int bad;
  if (fa)
    bad = launch_fa_prefill(group_of(c), (int)pitems.size(), c.n_kv_heads, q, kv->layer_base(layer),
                            (const SeqInfo*)(W + o_si), (const int32_t*)(W + o_bt), (const PrefillItem*)(W + o_pi), o,
                            scale_log2, st);
  else
    bad = launch_attn_generic(c.dtype, 0, cs.rows, n_seqs, c.n_q_heads, c.n_kv_heads, c.head_dim, q,
                              kv->layer_base(layer), (const SeqInfo*)(W + o_si), (const int32_t*)(W + o_bt), o,
                              1.0f / std::sqrt((float)c.head_dim), st);
  if (bad) return fail(PS_E_UNSUPPORTED, "attention configuration not supported");
  return last_launch_error();
  PS_CATCH
}

extern "C" ps_status ps_op_decode_plan(ps_kv* kv, int32_t n_seqs, const int32_t* seqs, int32_t split_pages,
                                       void* ws, size_t ws_bytes, void* stream) {
  PS_TRY CHECK_KV(kv);
  kv->dplan = DecodeAttnPlan{};
  const ps_layer_cfg& c = kv->cfg;
  if (!dec_ok(c)) return fail(PS_E_UNSUPPORTED, "split-K decode attention needs bf16, head_dim 128, G <= 16");
  if (split_pages < 0) return fail(PS_E_INVALID, "negative split_pages");
  CallSeqs cs;
  if (ps_status rc = plan_seqs(kv, n_seqs, seqs, nullptr, 1, cs)) return rc;
  Meta mt;
  DecodeAttnPlan pl;
  pl.o_si = mt.add(cs.si.data(), cs.si.size() * sizeof(SeqInfo));
  pl.o_bt = mt.add(cs.bt.data(), cs.bt.size() * 4);
  const int32_t sp = split_pages > 0 ? split_pages : choose_split_pages(cs.si, 0, c.n_kv_heads, PS_PHASE_ANSWER);
  DecodePlan dp = plan_decode(cs.si, 0, sp);
  if ((long)dp.items.size() > kMaxDecodeItems)
    return fail(PS_E_UNSUPPORTED, "more than 65535 attention work items: use larger split_pages");
  pl.o_di = mt.add(dp.items.data(), dp.items.size() * sizeof(DecodeItem));
  pl.o_pb = mt.add(dp.part_begin.data(), dp.part_begin.size() * 4);
  pl.o_pc = mt.add(dp.part_count.data(), dp.part_count.size() * 4);
  const size_t dq = (size_t)c.n_q_heads * c.head_dim;
  pl.off_po = mt.size();
  pl.off_pml = align_up(pl.off_po + (size_t)dp.n_parts * dq * 4, 256);
  pl.ws_need = align_up(pl.off_pml + (size_t)dp.n_parts * c.n_q_heads * 2 * 4, 256);
  if (ps_status rc = check_ws(ws, ws_bytes, pl.ws_need)) return rc;
  pl.ws = ws;
  pl.gen = kv->meta.generation();
  pl.n_seqs = n_seqs;
  pl.n_items = (int32_t)dp.items.size();
  if (n_seqs > 0) {
    void* host;
    const int slot = kv->staging.acquire(mt.size(), &host);
    if (slot < 0) return PS_E_HIP;
    std::memcpy(host, mt.buf.data(), mt.buf.size());
    if (ps_status rc = kv->staging.submit(slot, ws, mt.buf.size(), (hipStream_t)stream)) return rc;
  }
  kv->dplan = pl;
  return PS_OK;
  PS_CATCH
}

static ps_status decode_run(ps_kv* kv, int32_t layer, const void* q, void* o, void* ws, size_t ws_bytes,
                            int32_t max_workgroups, void* stream) {
  CHECK_KV(kv);
  if (ps_status rc = check_layer(kv, layer)) return rc;
  const DecodeAttnPlan& pl = kv->dplan;
  if (!pl.ws) return fail(PS_E_INVALID, "no decode attention plan on this handle");
  if (ws != pl.ws) return fail(PS_E_INVALID, "workspace differs from the planned one");
  if (pl.gen != kv->meta.generation())
    return fail(PS_E_INVALID, "the KV pool changed since the decode attention plan was made");
  if (ps_status rc = check_ws(ws, ws_bytes, pl.ws_need)) return rc;
  if (pl.n_seqs == 0) return PS_OK;
  if (!q || !o) return fail(PS_E_INVALID, "null pointer");
  if (ps_status rc = check_aligned({q, o})) return rc;
  const ps_layer_cfg& c = kv->cfg;
  char* W = (char*)ws;
  const float scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)c.head_dim));
  int bad = launch_decode_attn(group_of(c), pl.n_items, c.n_kv_heads, pl.n_seqs, q, kv->layer_base(layer),
                               (const SeqInfo*)(W + pl.o_si), (const int32_t*)(W + pl.o_bt),
                               (const DecodeItem*)(W + pl.o_di), (float*)(W + pl.off_po), (float*)(W + pl.off_pml),
                               (const int32_t*)(W + pl.o_pb), (const int32_t*)(W + pl.o_pc), o, scale_log2,
                               (hipStream_t)stream, max_workgroups);
  if (bad) return fail(PS_E_UNSUPPORTED, "decode attention configuration not supported");
  return last_launch_error();
}

extern "C" ps_status ps_op_decode_run(ps_kv* kv, int32_t layer, const void* q, void* o, void* ws, size_t ws_bytes,
                                      void* stream) {
  PS_TRY return decode_run(kv, layer, q, o, ws, ws_bytes, 0, stream);
  PS_CATCH
}

extern "C" ps_status ps_op_decode_run_capped(ps_kv* kv, int32_t layer, const void* q, void* o, void* ws,
                                             size_t ws_bytes, int32_t max_workgroups, void* stream) {
  PS_TRY if (max_workgroups < 1) return fail(PS_E_INVALID, "max_workgroups must be at least 1");
  return decode_run(kv, layer, q, o, ws, ws_bytes, max_workgroups, stream);
  PS_CATCH
}

extern "C" ps_status ps_op_decode_attention(ps_kv* kv, int32_t layer, int32_t n_seqs, const int32_t* seqs,
                                            const void* q, void* o, int32_t split_pages, void* ws, size_t ws_bytes,
                                            void* stream) {
  PS_TRY CHECK_KV(kv);
  if (ps_status rc = check_layer(kv, layer)) return rc;
  if (n_seqs > 0 && (!q || !o)) return fail(PS_E_INVALID, "null pointer");
  if (ps_status rc = ps_op_decode_plan(kv, n_seqs, seqs, split_pages, ws, ws_bytes, stream)) return rc;
  return ps_op_decode_run(kv, layer, q, o, ws, ws_bytes, stream);
  PS_CATCH
}
