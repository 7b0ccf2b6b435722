// Prefill (and chunked-prefill) causal attention over the paged KV cache,
// bf16 in, fp32 softmax, on the gfx950 matrix cores.
//
// A workgroup owns one 32-row query tile of one sequence and one KV head;
// its four waves are four query heads of that group (two workgroups per KV
// head when G = 8), so every K/V tile staged in LDS serves all of them (GQA
// reuse). Keys are walked in 32-key tiles (two pages) from position 0 up to
// the tile's last query position; the cached prefix of a chunked prefill is
// just the first pages of the walk.
//
// Both products are arranged so that softmax statistics never cross lanes:
//
//   S^T[key, q] = K[key, :] . Q[q, :]            (A = K rows, B = Q)
//   O^T[dim, q] += V^T[dim, key] P^T[key, q]      (A = V^T rows, B = P^T)
//
// With v_mfma_f32_32x32x16_bf16 a lane holds one query column of both S^T
// and O^T, so the online-softmax rescale is lane-local and the S^T
// accumulator, exponentiated and rounded to bf16, is already the B operand
// of the PV product. The V^T pages (dimension-major) make the A operand a
// contiguous 16-byte read.
//
// K and V^T tiles go from the pool straight into LDS by buffer DMA
// (buffer_load_dwordx4 ... lds, 1 KiB per wave instruction, no staging
// registers), double-buffered: the next tile's fills are issued before this
// tile's products and waited for at the one barrier per tile. DMA writes
// each instruction's 1 KiB contiguously, so bank spreading is by XOR
// swizzle rather than padding, and the K rows are stored in a permuted
// order (below) that makes P come out in the pool's key order.
//
// The per-score vector work is kept minimal. The softmax is invariant to
// the exponent base subtracted from a row's scores, so the base is not the
// running max: it is set from the row's true max only on the first tile
// and whenever this tile's row sum, computed anyway, shows the base stale
// (a sum past 2^32), so steady-state tiles take no max at all. The scale
// folds into one FMA per exponent; the row sum l is one packed bf16 dot
// product (v_dot2, against ones) per pair of P values, accumulated in
// fp32: the sum of exactly the bf16 P values the PV product uses, so
// V == 1 gives 1 to fp32 rounding, exactly 1 after the bf16 store. The
// half-wave max and sum exchanges are v_permlane32_swap.
//
// 32 KB of LDS and 150 registers per lane let three workgroups (three
// waves per SIMD) share a CU.
#include "common.h"
#include "launch.h"

#include <type_traits>

namespace ps {

namespace {
constexpr int kHd = 128;
constexpr int KT = 32;   // keys per tile (two pages, one per pair of waves)
constexpr int kQT = 32;  // query rows per workgroup tile (one 32-row block per wave)
}  // namespace

// One 16-byte pool->LDS fill per lane through a buffer resource: a wave
// instruction fills 1 KiB of LDS at `lds`, lane l landing at +16 l.
__device__ __forceinline__ void fa_dma16(__amdgpu_buffer_rsrc_t r, uint32_t voffset, bf16_t* lds) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds, 16, voffset, 0, 0, 0);
}

// Workgroup barrier that publishes this wave's pool->LDS fills and LDS
// writes: it waits for them first (vmcnt(0) lgkmcnt(0)). The fence of
// __syncthreads() alone does not order the fills, whose LDS writes are
// counted on vmcnt; without the wait a wave may pass the barrier before
// its fills land and another wave reads the stale slot.
__device__ __forceinline__ void fa_barrier() {
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
}

__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(3))) void fa_prefill_kernel(const bf16_t* __restrict__ q,
                                                         const bf16_t* __restrict__ pool,
                                                         const SeqInfo* __restrict__ si,
                                                         const int32_t* __restrict__ bt,
                                                         const PrefillItem* __restrict__ items,
                                                         bf16_t* __restrict__ o, int n_kv, int G, float scale_log2) {
  constexpr int NT = 256;
  constexpr int NPG = 2;
  constexpr int kKB = kPageTokens * kHd;  // elements of a page's K block (its V^T block follows)
  // K tile: 32 rows of 256 B; row r holds key 16 (r >> 4) + swap23(r & 15) (bits 2
  // and 3 exchanged, so that the S^T accumulator comes out with the keys of
  // each 16-key page in the order the PV product's B operand takes them:
  // lane half g holds keys 8g .. 8g + 7), its 16-byte chunk p holding dims
  // of chunk p ^ (r & 15).
  // V^T tile: per page, 128 dim rows of 32 B, 16-byte chunk q of row d
  // holding keys 8 (q ^ ((d >> 3) & 1)) .. + 8 of the page.
  __shared__ __attribute__((aligned(1024))) bf16_t sK0[KT * kHd];
  __shared__ __attribute__((aligned(1024))) bf16_t sK1[KT * kHd];
  __shared__ __attribute__((aligned(1024))) bf16_t sV0[KT * kHd];
  __shared__ __attribute__((aligned(1024))) bf16_t sV1[KT * kHd];

  const int hq = G / 4;
  const int kvh = blockIdx.y / hq;
  const PrefillItem it = items[blockIdx.x];
  const SeqInfo s = si[it.b];
  const int n_q = n_kv * G;
  const int t = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6), lane = t & 63;
  const int g = lane >> 5, c = lane & 31;
  const int head = kvh * G + (blockIdx.y % hq) * 4 + wave;
  const int qn = min(kQT, s.n_new - it.q_begin);
  const int qpos0 = s.kv_before + it.q_begin;
  const int n_keys = qpos0 + qn;
  const int kv_valid = s.kv_before + s.n_new;
  const int32_t* btr = bt + s.bt_off;
  const int n_tiles = (n_keys + KT - 1) / KT;
  const bf16_t* pool_h = pool + (long)kvh * (2L * kKB);
  const long page_stride = (long)n_kv * (2L * kKB);

  // DMA assignment: wave w fills page w >> 1 of each tile, half h = w & 1:
  // K rows 8h .. 8h + 7 (two 1 KiB fills of four rows) and V^T dims
  // 64h .. 64h + 63 (two fills of 32 dims).
  const int pg = wave >> 1, hh = wave & 1;
  uint32_t koff[2], voff[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int rr = 8 * hh + 4 * i + (lane >> 4), p = lane & 15;  // LDS row within the page
    const int tk = (rr & 3) | ((rr & 4) << 1) | ((rr & 8) >> 1);   // its token: bits 2, 3 swapped
    koff[i] = (uint32_t)(tk * kHd + ((p ^ rr) << 3)) * 2;
    const int d = 64 * hh + 32 * i + (lane >> 1), qq = lane & 1;
    voff[i] = (uint32_t)(kKB + d * kPageTokens + ((qq ^ ((d >> 3) & 1)) << 3)) * 2;
  }
  // page id of this wave's page in the tile at k0 (a scalar load, issued a
  // tile ahead of its use); pages past the written keys are never read
  auto page_id = [&](int k0) { return k0 + kPageTokens * pg < kv_valid ? btr[k0 / kPageTokens + pg] : 0; };
  auto issue = [&](int k0, int pid, bf16_t* dK, bf16_t* dV) {
    if (k0 + kPageTokens * pg >= kv_valid) return;  // page past the written keys: zeroed after landing
    const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<bf16_t*>(pool_h + (long)pid * page_stride), (short)0, (int)(2 * kKB * 2), 0x00020000);
    fa_dma16(r, koff[0], dK + (16 * pg + 8 * hh) * kHd);
    fa_dma16(r, koff[1], dK + (16 * pg + 8 * hh + 4) * kHd);
    fa_dma16(r, voff[0], dV + pg * kKB + (64 * hh) * kPageTokens);
    fa_dma16(r, voff[1], dV + pg * kKB + (64 * hh + 32) * kPageTokens);
  };
  // zero the V^T entries of keys at or past kv_valid in the tile at k0
  // (unwritten pool slots, or stale LDS for pages not filled)
  auto zero_tail = [&](int k0, bf16_t* dV) {
#pragma unroll
    for (int u0 = 0; u0 < 512; u0 += NT) {
      const int u = u0 + t;
      const int p = u >> 8, d = (u >> 1) & 127, qq = u & 1;
      const int kc = qq ^ ((d >> 3) & 1);
      const int valid = kv_valid - (k0 + kPageTokens * p + 8 * kc);
      if (valid >= 8) continue;
      uint4* ptr = (uint4*)(dV + p * kKB + d * kPageTokens + qq * 8);
      uint4 w = *ptr;
      uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (j >= valid) ws[j >> 1] &= (j & 1) ? 0x0000ffffu : 0xffff0000u;
      *ptr = make_uint4(ws[0], ws[1], ws[2], ws[3]);
    }
  };

  bf16x8_t qf[8];
  {
    int r = min(c, qn - 1);
    const bf16_t* qp = q + ((long)(s.row_start + it.q_begin + r) * n_q + head) * kHd + 8 * g;
#pragma unroll
    for (int kk = 0; kk < 8; ++kk) qf[kk] = __builtin_bit_cast(bf16x8_t, *(const uint4*)(qp + 16 * kk));
  }
  f32x16_t oacc[4];
#pragma unroll
  for (int db = 0; db < 4; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[db][r] = 0.f;
  float lsum = 0.f;
  float m = -INFINITY, mb = -INFINITY;  // row max behind the exponent base (set by the first tile), and m scale
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  const bf16x2_t ones2 = {(__bf16)1.0f, (__bf16)1.0f};
  // lane-constant LDS byte offsets of the operand reads
  const uint32_t kread = (uint32_t)(c * kHd * 2 + ((g ^ (c & 15)) << 4));        // ^ (32 kk) per chunk
  const uint32_t vread = (uint32_t)(c * kPageTokens * 2 + ((g ^ ((c >> 3) & 1)) << 4));  // + page, dim block

  // one key tile: K, V hold it; the next tile's fills go to nK, nV
  int pid_next = n_tiles > 1 ? page_id(KT) : 0;
  // `firstc`: std::true_type for the walk's first tile, which sets the base
  auto tile = [&](int kt, const bf16_t* K, const bf16_t* V, bf16_t* nK, bf16_t* nV, auto firstc) {
    constexpr bool FIRST = decltype(firstc)::value;
    const int k0 = kt * KT;
    if (kt + 1 < n_tiles) {
      issue(k0 + KT, pid_next, nK, nV);
      if (kt + 2 < n_tiles) pid_next = page_id(k0 + 2 * KT);
    }
    f32x16_t sacc;
#pragma unroll
    for (int r = 0; r < 16; ++r) sacc[r] = 0.f;
#pragma unroll
    for (int kk = 0; kk < 8; ++kk) {
      const bf16x8_t a = __builtin_bit_cast(bf16x8_t, *(const uint4*)((const char*)K + (kread ^ (32 * kk))));
      sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[kk], sacc, 0, 0, 0);
    }
    // padding columns (c >= qn) take the last row's keys: rows past it may
    // hold unwritten pool slots
    const int qpos = qpos0 + min(c, qn - 1);
    if (k0 + KT - 1 > qpos0) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = k0 + 16 * (r >> 3) + 8 * g + 4 * ((r >> 2) & 1) + (r & 3);
        if (key > qpos) sacc[r] = -INFINITY;
      }
    }
    // P = 2^(s scale - mb) against the row's exponent base mb, and this
    // lane's partial row sum of the bf16 P values. The first tile sets the
    // base from its own row max (key 0 is visible to every query row, so that
    // max is finite). After it, the sum doubles as the test of the base: past
    // 2^32 (or infinite or NaN, where an exponent overflowed) the tile takes
    // the slow path, which takes the row's true max over the tile, rescales O
    // and l to it and redoes the exponentials. While the base stands no max
    // is taken at all.
    uint32_t pk[8];
    auto exps = [&]() __attribute__((always_inline)) {
#pragma unroll
      for (int i = 0; i < 8; ++i)
        pk[i] = pack_bf2(__builtin_amdgcn_exp2f(fmaf(sacc[2 * i], scale_log2, -mb)),
                         __builtin_amdgcn_exp2f(fmaf(sacc[2 * i + 1], scale_log2, -mb)));
      float lt = 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) lt = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, pk[i]), ones2, lt, false);
      return lt;
    };
    auto row_max = [&]() __attribute__((always_inline)) {
      float mx = sacc[0];
#pragma unroll
      for (int r = 1; r < 16; ++r) mx = fmaxf(mx, sacc[r]);
      // the other half's max (lane l +- 32) without an LDS round trip
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
      return fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
    };
    float lt;
    if constexpr (FIRST) {
      m = row_max();
      mb = m * scale_log2;
      lt = exps();
    } else {
      lt = exps();
      if (__any(!(lt <= 0x1p32f))) {
        const float m_new = fmaxf(m, row_max());
        const float alpha = __builtin_amdgcn_exp2f((m - m_new) * scale_log2);
#pragma unroll
        for (int db = 0; db < 4; ++db)
#pragma unroll
          for (int r = 0; r < 16; ++r) oacc[db][r] *= alpha;
        lsum *= alpha;
        m = m_new;
        mb = m * scale_log2;
        lt = exps();
      }
    }
    lsum += lt;
#pragma unroll
    for (int kk2 = 0; kk2 < NPG; ++kk2) {
      const bf16x8_t bp = __builtin_bit_cast(bf16x8_t, make_uint4(pk[4 * kk2], pk[4 * kk2 + 1], pk[4 * kk2 + 2], pk[4 * kk2 + 3]));
#pragma unroll
      for (int db = 0; db < 4; ++db) {
        const bf16x8_t a = __builtin_bit_cast(
            bf16x8_t, *(const uint4*)((const char*)V + kk2 * kKB * 2 + db * 32 * kPageTokens * 2 + vread));
        oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, bp, oacc[db], 0, 0, 0);
      }
    }
    fa_barrier();  // this wave's fills of the next tile landed; every wave is done with this tile
    if (kt + 1 < n_tiles && k0 + 2 * KT > kv_valid) {
      zero_tail(k0 + KT, nV);
      fa_barrier();
    }
  };

  issue(0, page_id(0), sK0, sV0);
  fa_barrier();
  if (KT > kv_valid) {
    zero_tail(0, sV0);
    fa_barrier();
  }
  // tile t sits in slot t & 1; the first tile is peeled (it sets the base)
  tile(0, sK0, sV0, sK1, sV1, std::true_type{});
  for (int kt = 1; kt < n_tiles; kt += 2) {
    tile(kt, sK1, sV1, sK0, sV0, std::false_type{});
    if (kt + 1 < n_tiles) tile(kt + 1, sK0, sV0, sK1, sV1, std::false_type{});
  }

  {
    const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(lsum), __float_as_uint(lsum), false, false);
    const float l = __uint_as_float(sw[0]) + __uint_as_float(sw[1]);  // lower half's part + upper half's
    if (c < qn) {
      const float inv = 1.f / l;
      bf16_t* op = o + ((long)(s.row_start + it.q_begin + c) * n_q + head) * kHd;
#pragma unroll
      for (int db = 0; db < 4; ++db)
#pragma unroll
        for (int rb = 0; rb < 4; ++rb) {
          const int dim = 32 * db + 8 * rb + 4 * g;
          uint2 w = make_uint2(pack_bf2(oacc[db][4 * rb] * inv, oacc[db][4 * rb + 1] * inv),
                               pack_bf2(oacc[db][4 * rb + 2] * inv, oacc[db][4 * rb + 3] * inv));
          *(uint2*)(op + dim) = w;
        }
    }
  }
}

int fa_query_tile() { return kQT; }

int launch_fa_prefill(int G, int n_items, int n_kv, const void* q, const void* pool_layer, const SeqInfo* si,
                      const int32_t* bt, const PrefillItem* items, void* o, float scale_log2, hipStream_t st) {
  if (n_items == 0) return 0;
  if (G % 4 != 0) return -1;
  dim3 grid(n_items, n_kv * (G / 4));
  hipLaunchKernelGGL(fa_prefill_kernel, grid, dim3(256), 0, st, (const bf16_t*)q, (const bf16_t*)pool_layer, si, bt,
                     items, (bf16_t*)o, n_kv, G, scale_log2);
  return 0;
}

}  // namespace ps
