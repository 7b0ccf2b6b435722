// Prefill (and chunked-prefill) causal attention over the paged KV cache,
// bf16 in, fp32 softmax, on the gfx950 matrix cores.
//
// A workgroup owns one 32-row query tile (32 * kFaQB rows, kFaQB = 1) of one
// sequence and one KV head; its waves are four query heads of that group
// (two workgroups per KV head when G = 8), so every K/V tile staged
// in LDS serves all of them (GQA reuse). Keys are walked in 32-key tiles
// (two pages) from position 0 up to the tile's last query position; the
// cached prefix of a chunked prefill is just the first pages of the walk.
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
// contiguous read. LDS rows are padded (272 B for K, 80 B for V^T) so the
// 16-byte operand reads of 16 consecutive lanes hit disjoint banks.
//
// The matrix cores are busy about a third of the time: each MFMA waits on
// its own LDS operand read and the softmax sits between the two products.
// The per-score vector work is kept minimal: the running max is taken on
// raw scores and the scale folds into one FMA per exponent, the output is
// rescaled only when a row's max outgrows the exponent base by 2^8, and the row sum
// l is one packed bf16 dot product (v_dot2, against ones) per pair of P values,
// accumulated in fp32: the sum of exactly the bf16 P values the PV product
// uses, so V == 1 gives 1 to fp32 rounding, exactly 1 after the bf16 store.
//
// The short tiles keep the LDS footprint at 45 KB and the registers at 168
// per lane, so three workgroups (three waves per SIMD) share a CU; their
// interleaving hides the LDS and global latency one wave cannot.
#include "common.h"
#include "launch.h"

namespace ps {

namespace {
constexpr int kHd = 128;
constexpr int kFaKT = 32;            // keys per tile (two pages)
constexpr int kPageCache = 2048;     // page ids cached in LDS (32768 positions)
constexpr int kFaQB = 1;             // query blocks of 32 rows per wave (1: lower register pressure, 2.3x faster than 2)
}  // namespace

// Four waves = four query heads of one KV group per workgroup; groups of 8
// heads use two workgroups per KV head. K/V tiles are double-buffered: the
// next tile's global loads are issued into registers before the current
// tile's products, and written to the other LDS buffer after them, so one
// barrier per tile suffices and load latency hides behind the MFMAs.
template <int QB, int KT>  // 32-row query blocks per wave (query tile 32 * QB rows); keys per tile
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(3))) void fa_prefill_kernel(const bf16_t* __restrict__ q,
                                                         const bf16_t* __restrict__ pool,
                                                         const SeqInfo* __restrict__ si,
                                                         const int32_t* __restrict__ bt,
                                                         const PrefillItem* __restrict__ items,
                                                         bf16_t* __restrict__ o, int n_kv, int G, float scale_log2) {
  constexpr int NT = 256;
  constexpr int kQT = 32 * QB;
  constexpr int NPG = KT / kPageTokens;  // pages per key tile
  constexpr int NKB = KT / 32;           // 32-key blocks per key tile
  constexpr int KRow = kHd + 8;          // padded K row (elements)
  constexpr int VRow = KT + 8;           // padded V^T row (elements)
  static_assert(KT % 32 == 0 && (NPG == 2 || NPG == 4) && kPageCache % NPG == 0, "key tile");
  __shared__ __attribute__((aligned(16))) bf16_t sK[2][KT * KRow];
  __shared__ __attribute__((aligned(16))) bf16_t sV[2][kHd * VRow];
  __shared__ __attribute__((aligned(16))) int32_t sPage[kPageCache];  // a window of the walk's page ids

  const int hq = G / 4;  // workgroups per KV head
  const int kvh = blockIdx.y / hq;
  const PrefillItem it = items[blockIdx.x];
  const SeqInfo s = si[it.b];
  const int n_q = n_kv * G;
  const int t = threadIdx.x;
  const int wave = t >> 6, lane = t & 63;
  const int g = lane >> 5, c = lane & 31;
  const int head = kvh * G + (blockIdx.y % hq) * 4 + wave;
  const int qn = min(kQT, s.n_new - it.q_begin);       // valid rows in this tile
  const int qpos0 = s.kv_before + it.q_begin;           // position of tile row 0
  const int n_keys = qpos0 + qn;                        // keys 0 .. last query position
  const int kv_valid = s.kv_before + s.n_new;
  const int32_t* btr = bt + s.bt_off;
  // every page a tile load can touch: keys below kv_valid inside the walk's
  // n_tiles key tiles (the last tile may reach past the last query)
  const int n_tiles = (n_keys + KT - 1) / KT;
  const int n_pages_walk = min((kv_valid + kPageTokens - 1) / kPageTokens, n_tiles * NPG);
  // page ids of the walk, cached in LDS in windows of kPageCache pages
  // (a tile's pages never straddle a window: kPageCache is a multiple of NPG)
  int win = 0;  // first page of the cached window
  auto fill_pages = [&]() {
    for (int i = t; i < min(n_pages_walk - win, kPageCache); i += NT) sPage[i] = btr[win + i];
  };
  fill_pages();
  __syncthreads();
  // page ids of the tile at key k0 (pages k0/16 ..), one LDS read
  auto tile_pages = [&](int k0, int (&pid)[NPG]) {
    const int* sp = &sPage[k0 / kPageTokens - win];
    if constexpr (NPG == 4) {
      const int4 pp = *(const int4*)sp;
      pid[0] = __builtin_amdgcn_readfirstlane(pp.x);
      pid[1] = __builtin_amdgcn_readfirstlane(pp.y);
      pid[2] = __builtin_amdgcn_readfirstlane(pp.z);
      pid[3] = __builtin_amdgcn_readfirstlane(pp.w);
    } else {
      const int2 pp = *(const int2*)sp;
      pid[0] = __builtin_amdgcn_readfirstlane(pp.x);
      pid[1] = __builtin_amdgcn_readfirstlane(pp.y);
    }
  };
  const long kvh_off = (long)kvh * (2L * kPageTokens * kHd);
  const long page_stride = (long)n_kv * (2L * kPageTokens * kHd);

  // Q^T operand: lane (g, c) holds Q[row 32cb + c][16kk + 8g .. +8]
  bf16x8_t qf[QB][8];
#pragma unroll
  for (int cb = 0; cb < QB; ++cb) {
    int r = min(32 * cb + c, qn - 1);
    const bf16_t* qp = q + ((long)(s.row_start + it.q_begin + r) * n_q + head) * kHd + 8 * g;
#pragma unroll
    for (int kk = 0; kk < 8; ++kk) qf[cb][kk] = __builtin_bit_cast(bf16x8_t, *(const uint4*)(qp + 16 * kk));
  }

  // oacc[cb][db]: O^T dims 32 db + ...; lsum: this lane's half of l (keys with offset 4g)
  f32x16_t oacc[QB][4];
  float lsum[QB];
#pragma unroll
  for (int cb = 0; cb < QB; ++cb) lsum[cb] = 0.f;
#pragma unroll
  for (int cb = 0; cb < QB; ++cb)
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) oacc[cb][db][r] = 0.f;
  float m[QB];  // exponent base of each row block (raw, unscaled score units)
#pragma unroll
  for (int cb = 0; cb < QB; ++cb) m[cb] = -INFINITY;
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  const bf16x2_t ones2 = {(__bf16)1.0f, (__bf16)1.0f};

  // staging assignment: load i of thread t covers page i of the tile: K row
  // t / 16, 16-byte chunk t % 16; V^T dim t / 2, keys 8 (t % 2) .. + 8. The
  // page ids are workgroup-uniform (scalar), the per-lane offsets fixed.
  const int koff = (t >> 4) * kHd + (t & 15) * 8;
  const int voff = kPageTokens * kHd + (t >> 1) * kPageTokens + (t & 1) * 8;
  uint4 rk[NPG], rv[NPG];
  auto gload = [&](int k0) {
    int pids[NPG];
    tile_pages(k0, pids);
    if (k0 + KT <= kv_valid) {  // every key of the tile written: plain loads
#pragma unroll
      for (int i = 0; i < NPG; ++i) {
        const bf16_t* base = pool + (long)pids[i] * page_stride + kvh_off;
        rk[i] = *(const uint4*)(base + koff);
        rv[i] = *(const uint4*)(base + voff);
      }
      return;
    }
#pragma unroll
    for (int i = 0; i < NPG; ++i) {
      const int p0 = k0 + i * kPageTokens;  // first position of page i
      rk[i] = make_uint4(0, 0, 0, 0);
      rv[i] = make_uint4(0, 0, 0, 0);
      if (p0 >= kv_valid) continue;
      const bf16_t* base = pool + (long)pids[i] * page_stride + kvh_off;
      if (p0 + (t >> 4) < kv_valid) rk[i] = *(const uint4*)(base + koff);
      uint4 w = *(const uint4*)(base + voff);
      // zero V^T entries of keys past the written length
      const int valid = kv_valid - p0 - (t & 1) * 8;
      if (valid < 8) {
        uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
        for (int j = 0; j < 8; ++j)
          if (j >= valid) ws[j >> 1] &= (j & 1) ? 0x0000ffffu : 0xffff0000u;
        w = make_uint4(ws[0], ws[1], ws[2], ws[3]);
      }
      rv[i] = w;
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < NPG; ++i) {
      *(uint4*)(&sK[buf][(16 * i + (t >> 4)) * KRow + (t & 15) * 8]) = rk[i];
      // half hf = keys 8hf..8hf+7; stored per page as [0-3][8-11][4-7][12-15]
      const int dim = t >> 1, hf = t & 1;
      bf16_t* dst = &sV[buf][dim * VRow + i * kPageTokens];
      *(uint2*)(dst + hf * 4) = make_uint2(rv[i].x, rv[i].y);
      *(uint2*)(dst + 8 + hf * 4) = make_uint2(rv[i].z, rv[i].w);
    }
  };

  gload(0);
  lstore(0);
  __syncthreads();
  for (int kt = 0; kt < n_tiles; ++kt) {
    const int k0 = kt * KT;
    const int buf = kt & 1;
    if (kt + 1 < n_tiles) {
      if ((k0 + KT) / kPageTokens - win >= kPageCache) {  // the next tile starts a new window
        win += kPageCache;  // every wave is past its last read of the old window (barrier below)
        fill_pages();
        __syncthreads();
      }
      gload(k0 + KT);
    }
    const bf16_t* K = sK[buf];
    const bf16_t* V = sV[buf];
    bool act[QB];  // block 0 always has a row (qn >= 1); a compile-time true keeps its products branch-free
#pragma unroll
    for (int cb = 0; cb < QB; ++cb) act[cb] = cb == 0 || 32 * cb < qn;
    // S^T per 32-key block and row block, each K fragment read once
    f32x16_t sacc[NKB][QB];
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
      for (int cb = 0; cb < QB; ++cb)
#pragma unroll
        for (int r = 0; r < 16; ++r) sacc[kb][cb][r] = 0.f;
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
      for (int kk = 0; kk < 8; ++kk) {
        const bf16x8_t a = __builtin_bit_cast(bf16x8_t, *(const uint4*)(K + (32 * kb + c) * KRow + 16 * kk + 8 * g));
#pragma unroll
        for (int cb = 0; cb < QB; ++cb)
          if (act[cb]) sacc[kb][cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[cb][kk], sacc[kb][cb], 0, 0, 0);
      }
    // sacc[kb][cb][r] = score(key 32kb + 8(r/4) + 4g + r%4, query 32cb + c);
    // mask only on tiles that reach past the block's first query position
    uint32_t pk[NKB][QB][8];
#pragma unroll
    for (int cb = 0; cb < QB; ++cb) {
      if (!act[cb]) continue;
      const int qpos = qpos0 + 32 * cb + c;
      if (k0 + KT - 1 > qpos0 + 32 * cb) {
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int key = k0 + 32 * kb + 8 * (r >> 2) + 4 * g + (r & 3);
            if (key > qpos) sacc[kb][cb][r] = -INFINITY;
          }
      }
      float mx = sacc[0][cb][0];
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sacc[kb][cb][r]);
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      // The exponent base m moves only when some row's max exceeds it by
      // more than 8 in the exp2 domain (so P <= 2^8); O and l carry the
      // same base, which cancels in O / l. Rows rarely cross the margin
      // after the first tiles, so the 80-register rescale is mostly skipped.
      // The first tile always moves it (m = -inf); key 0 is in every row's
      // first tile, so m is finite from then on.
      if (__any((mx - m[cb]) * scale_log2 > 8.f)) {
        const float m_new = fmaxf(m[cb], mx);
        const float alpha = __builtin_amdgcn_exp2f((m[cb] - m_new) * scale_log2);  // lane-local factor
#pragma unroll
        for (int db = 0; db < 4; ++db)
#pragma unroll
          for (int r = 0; r < 16; ++r) oacc[cb][db][r] *= alpha;
        lsum[cb] *= alpha;
        m[cb] = m_new;
      }
      const float mb = m[cb] * scale_log2;
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
        for (int i = 0; i < 8; ++i)
          pk[kb][cb][i] = pack_bf2(__builtin_amdgcn_exp2f(fmaf(sacc[kb][cb][2 * i], scale_log2, -mb)),
                                   __builtin_amdgcn_exp2f(fmaf(sacc[kb][cb][2 * i + 1], scale_log2, -mb)));
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
        for (int i = 0; i < 8; ++i)
          lsum[cb] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, pk[kb][cb][i]), ones2, lsum[cb], false);
    }
    // O^T += V^T P^T per page (16 keys) and row block, each V fragment read once
#pragma unroll
    for (int kk2 = 0; kk2 < NPG; ++kk2) {
      const int kb = kk2 >> 1, hl = kk2 & 1;
      bf16x8_t bp[QB];
#pragma unroll
      for (int cb = 0; cb < QB; ++cb)
        bp[cb] = __builtin_bit_cast(bf16x8_t, make_uint4(pk[kb][cb][4 * hl], pk[kb][cb][4 * hl + 1],
                                                         pk[kb][cb][4 * hl + 2], pk[kb][cb][4 * hl + 3]));
#pragma unroll
      for (int db = 0; db < 4; ++db) {
        const bf16x8_t a = __builtin_bit_cast(
            bf16x8_t, *(const uint4*)(V + (32 * db + c) * VRow + kk2 * kPageTokens + 8 * g));
#pragma unroll
        for (int cb = 0; cb < QB; ++cb)
          if (act[cb]) oacc[cb][db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, bp[cb], oacc[cb][db], 0, 0, 0);
      }
    }
    if (kt + 1 < n_tiles) lstore(buf ^ 1);
    __syncthreads();
  }

  // ---- normalise and store: lane holds query c, dims 32db + 8(r/4) + 4g + r%4
#pragma unroll
  for (int cb = 0; cb < QB; ++cb) {
    const float l = lsum[cb] + __shfl_xor(lsum[cb], 32);
    const int r0 = 32 * cb + c;
    if (r0 >= qn) continue;
    const float inv = 1.f / l;
    bf16_t* op = o + ((long)(s.row_start + it.q_begin + r0) * n_q + head) * kHd;
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int rb = 0; rb < 4; ++rb) {
        const int dim = 32 * db + 8 * rb + 4 * g;
        uint2 w = make_uint2(pack_bf2(oacc[cb][db][4 * rb] * inv, oacc[cb][db][4 * rb + 1] * inv),
                             pack_bf2(oacc[cb][db][4 * rb + 2] * inv, oacc[cb][db][4 * rb + 3] * inv));
        *(uint2*)(op + dim) = w;
      }
  }
}

int fa_query_tile() { return 32 * kFaQB; }

template <int QB>
int launch_fa_prefill_qb(int G, int n_items, int n_kv, const void* q, const void* pool_layer, const SeqInfo* si,
                         const int32_t* bt, const PrefillItem* items, void* o, float scale_log2, hipStream_t st) {
  if (n_items == 0) return 0;
  if (G % 4 != 0) return -1;
  dim3 grid(n_items, n_kv * (G / 4));
  hipLaunchKernelGGL((fa_prefill_kernel<QB, kFaKT>), grid, dim3(256), 0, st, (const bf16_t*)q, (const bf16_t*)pool_layer, si,
                     bt, items, (bf16_t*)o, n_kv, G, scale_log2);
  return 0;
}

int launch_fa_prefill(int G, int n_items, int n_kv, const void* q, const void* pool_layer, const SeqInfo* si,
                      const int32_t* bt, const PrefillItem* items, void* o, float scale_log2, hipStream_t st) {
  return launch_fa_prefill_qb<kFaQB>(G, n_items, n_kv, q, pool_layer, si, bt, items, o, scale_log2, st);
}

}  // namespace ps
