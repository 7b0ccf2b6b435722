// GEMMs of the layer: C = epilogue(A W^T), A [M, K] row-major, W [N, K]
// (the nn.Linear orientation) stored in 64x64 tiles: tile (i, j) covers rows
// 64i.. and columns 64j.., sits at tile index i * ceil(K/64) + j, and is
// row-major inside (64 rows of 64 elements). Every 64-row by 64-k slab a
// workgroup streams is then one contiguous 8 KiB (bf16) block of HBM rather
// than 64 strided 128-byte pieces. fp32 accumulation (gfx950).
//
//  * gemm_tile_kernel: prefill-sized M. 256x256 workgroup tile, four waves
//    of 128x128 (one per SIMD), v_mfma_f32_32x32x16_bf16 with accumulators
//    in AGPRs, 64-k stages in two XOR-swizzled LDS slots (128 KiB) filled
//    by direct global->LDS loads spread over the stage. MFMA-bound.
//  * gemm_skinny_kernel: decode-sized M (<= 64). Streams W once from HBM
//    with 16-byte loads, one 16-column MFMA block per wave, activations
//    staged in LDS and shared by the workgroup's four waves; K may be split
//    across workgroups, fp32 partials then reduced in split order by
//    gemm_reduce_kernel. HBM-bound (AI = M FLOP/byte).
//  * gemm_f32_kernel: fp32 layers, 64x64 register-blocked vector FMA.
//
// Epilogues: store, residual add (C = R + A W^T) and SwiGLU (W rows
// interleaved gate/up in blocks of 32; C[:, j] = silu(gate_j) * up_j).
#include "common.h"
#include "launch.h"

#include <mutex>
#include <type_traits>

namespace ps {

__device__ __forceinline__ float silu_f(float x) { return x / (1.f + expf(-x)); }
// silu on the hardware exp2 and reciprocal (v_exp_f32, v_rcp_f32): a few
// fp32 ulp, far below the bf16 rounding of the GEMM operands; four vector
// instructions instead of the ~30 of expf and an IEEE divide, which matter
// in an epilogue that no matrix work overlaps. x -> -inf gives -0, x -> inf
// gives x.
__device__ __forceinline__ float silu_fast(float x) {
  return x * __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(x * -1.4426950408889634f));
}

template <typename T> __device__ __forceinline__ float ld_elt(const T* p, long i);
template <> __device__ __forceinline__ float ld_elt<float>(const float* p, long i) { return p[i]; }
template <> __device__ __forceinline__ float ld_elt<bf16_t>(const bf16_t* p, long i) { return bf2f(p[i]); }
template <typename T> __device__ __forceinline__ void st_elt(T* p, long i, float v);
template <> __device__ __forceinline__ void st_elt<float>(float* p, long i, float v) { p[i] = v; }
template <> __device__ __forceinline__ void st_elt<bf16_t>(bf16_t* p, long i, float v) { p[i] = f2bf(v); }

// ================================================================== helpers
// One 16-byte global->LDS fill per lane through a buffer resource
// (buffer_load_dwordx4 ... lds): a wave instruction fills 1 KiB of LDS, lane
// l landing at +16 l; `voffset` is the lane's byte offset from the resource
// base. The compiler counts this form on vmcnt alone, so LDS reads issued
// around it keep exact lgkmcnt waits (around the FLAT global_load_lds form
// it waits for every outstanding LDS read before each use of a fragment).
__device__ __forceinline__ void load_lds16_buf(__amdgpu_buffer_rsrc_t r, uint32_t voffset, bf16_t* lds) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds, 16, voffset, 0, 0, 0);
}
// The same with a wave-uniform byte offset in the scalar offset operand: a
// per-stage step added there costs no vector address arithmetic.
__device__ __forceinline__ void load_lds16_buf_so(__amdgpu_buffer_rsrc_t r, uint32_t voffset, uint32_t soffset,
                                                  bf16_t* lds) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds, 16, voffset, soffset, 0, 0);
}
// The same with the non-temporal hint (cache policy bit 1), for data read
// exactly once per call (decode weight streams).
__device__ __forceinline__ void load_lds16_buf_nt(__amdgpu_buffer_rsrc_t r, uint32_t voffset, bf16_t* lds) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds, 16, voffset, 0, 0, 2);
}
// Raw (stride 0) buffer resource over `bytes` bytes from `base`; loads past
// the end return zero.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

// s_waitcnt vmcnt(n) lgkmcnt(0): this wave's global->LDS fills older than
// its n most recent have landed, and its own LDS reads have returned.
template <int N>
__device__ __forceinline__ void wait_vmcnt_lgkm0() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4));
}

// Workgroup barrier without the release/acquire fences of __syncthreads():
// those wait for every outstanding global->LDS fill (vmcnt(0)) and would
// collapse a ring deeper than two stages. Callers wait explicitly first; the
// memory clobber keeps LDS accesses on their side of the barrier.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_barrier" ::: "memory"); }

// The same barrier pinned in the instruction schedule: register-only work
// (MFMAs) may not move across it either.
__device__ __forceinline__ void lds_barrier_pinned() {
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("s_barrier" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
}

// f(std::integral_constant<int, i>) for i = B .. E-1, unrolled at compile
// time (register arrays indexed by i stay in registers).
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

// ====================================================================== tile
// Prefill-sized M. Workgroup tile 256 x 256, four waves of 128 x 128 (one
// per SIMD), v_mfma_f32_32x32x16_bf16 with the 256 accumulators per lane in
// AGPRs. K runs in 64-wide stages through two LDS slots (128 KiB) filled by
// global->LDS DMA (buffer form); LDS rows are 128 B, their 16-byte chunks
// XOR-swizzled by (row / 2) % 8 so that the operand reads of 16 consecutive
// rows hit 16 distinct bank groups (the DMA lane addresses are chosen so
// that the linear fill lands swizzled).
//
// Schedule of stage st (slot st & 1), four 16-k slices of 16 MFMAs each.
// Every slice interleaves with its MFMAs:
//  * the reads of the next slice's eight fragments, one after each of the
//    first eight MFMAs, in the order the next slice first uses them
//    (a0 b0 b1 b2 b3 a1 a2 a3), so its MFMAs wait only for their own;
//  * DMA instructions, one after every other MFMA from the second: in
//    slices 0 and 1 the rest of stage st+1, in slice 3 the first part of
//    stage st+2 into slot st & 1.
// After slice 2: wait for stage st+1 and this stage's reads, one barrier
// (slot st & 1 is free from there, and slice 3 reads stage st+1's first
// fragments). Issued in bursts, DMA or reads back up the address unit and
// the LDS queue and stall the waves' instruction streams. The split over
// slices 3, 0, 1 is 7 / 7 / 2: loads issued in slice 1 have only a slice and
// a half to land before that wait, which an L2 miss outlasts (6 / 5 / 5 was
// 2% slower on the gate_up shape).
namespace tile {
constexpr int BM = 256, BN = 256, BK = 64, NT = 256, WT = 128;
constexpr int CPR = BK / 8, RPL = 64 / CPR;                         // 8 chunks per row, 8 rows per DMA
constexpr int A_ELTS = BM * BK, STAGE = (BM + BN) * BK;             // bf16 elements
constexpr int A_LOADS = BM / RPL / 4, B_LOADS = BN / RPL / 4, LOADS = A_LOADS + B_LOADS;  // per wave
constexpr int Q = WT / 32;                                           // 4 x 4 blocks of 32 x 32
constexpr int D3 = 7, D0 = 7, D1 = LOADS - D3 - D0;                  // DMA split over slices 3, 0, 1
constexpr int DMA_AT = 1, DMA_EVERY = 2;                             // after MFMAs 1, 3, 5, ...
static_assert(DMA_AT + (D3 - 1) * DMA_EVERY < Q * Q && DMA_AT + (D0 - 1) * DMA_EVERY < Q * Q &&
                  DMA_AT + (D1 - 1) * DMA_EVERY < Q * Q, "DMA slots in a slice");
constexpr size_t LDS_BYTES = 2 * (size_t)STAGE * 2;
__device__ __forceinline__ int swz(int row, int ch) { return row * BK + ((ch ^ ((row >> 1) & 7)) << 3); }
}  // namespace tile

template <int EPI, typename TR, typename TC>
__global__ __launch_bounds__(256) void gemm_tile_kernel(const bf16_t* __restrict__ A, const bf16_t* __restrict__ W,
                                                        const TR* __restrict__ R, TC* __restrict__ C, int M, int N,
                                                        int K, int tiles_n, int group, int splits) {
  using namespace tile;
  extern __shared__ __attribute__((aligned(16))) bf16_t smem[];

  // XCD-aware tile order: consecutive workgroup ids go round-robin over the
  // 8 XCDs; give each XCD a contiguous range of tiles, walked in groups of
  // `group` tile-rows across N, so that tiles sharing A and W panels meet in
  // the same L2.
  // With splits > 1 (EPI 0, fp32 C) the grid holds every tile once per K
  // split, split-major: split s covers stages [s T / splits, (s + 1) T /
  // splits) and stores its partial at C + s M N.
  const int nwg = gridDim.x;
  int id = blockIdx.x;
  if ((nwg & 7) == 0) id = (id & 7) * (nwg >> 3) + (id >> 3);
  const int n_tiles = nwg / splits;
  const int ks = id / n_tiles;
  id -= ks * n_tiles;
  const int tiles_m = n_tiles / tiles_n;
  const int group_sz = group * tiles_n;
  const int first_m = (id / group_sz) * group;
  const int gm = min(group, tiles_m - first_m);
  const int tm = first_m + (id % group_sz) % gm;
  const int tn = (id % group_sz) / gm;
  const int m0 = tm * BM, n0 = tn * BN;

  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int wm = wave >> 1, wn = wave & 1;
  // DMA sources: buffer resources at the tile's A rows and W blocks, 32-bit
  // lane byte offsets (rows past M read row M-1, results unused)
  const int lrow = lane / CPR, lpos = lane % CPR;
  uint32_t aoff[A_LOADS], boff[B_LOADS];
#pragma unroll
  for (int i = 0; i < A_LOADS; ++i) {
    const int row = (wave * A_LOADS + i) * RPL + lrow;
    aoff[i] = ((uint32_t)(min(m0 + row, M - 1) - m0) * K + (lpos ^ ((row >> 1) & 7)) * 8) * 2;
  }
#pragma unroll
  for (int i = 0; i < B_LOADS; ++i) {  // tiled W: rows of 64-row block row/64, k-tile added per stage
    const int row = (wave * B_LOADS + i) * RPL + lrow;
    boff[i] = ((uint32_t)(row >> 6) * (K / 64) * kWTileElts + (row & 63) * 64 + (lpos ^ ((row >> 1) & 7)) * 8) * 2;
  }
  static_assert(BK == kWTile, "one W tile per stage");
  const __amdgpu_buffer_rsrc_t rA = buffer_rsrc(A + (long)m0 * K, (uint32_t)min(M - m0, BM) * K * 2);
  const __amdgpu_buffer_rsrc_t rW =
      buffer_rsrc(W + (long)(n0 >> 6) * (K / 64) * kWTileElts, (uint32_t)(BN / 64) * (K / 64) * kWTileElts * 2);
  const int T_all = K / BK;
  const int st0 = ks * T_all / splits, T = (ks + 1) * T_all / splits - st0;  // this workgroup's stages
  // DMA instruction l (0..LOADS-1) of stage s into slot dslot (= s & 1);
  // the stage's step rides in the scalar offset
  auto dma = [&](int s, int dslot, int l) __attribute__((always_inline)) {
    bf16_t* st = smem + dslot * STAGE;
    if (l < A_LOADS)
      load_lds16_buf_so(rA, aoff[l], (s + st0) * BK * 2, st + (wave * A_LOADS + l) * RPL * BK);
    else
      load_lds16_buf_so(rW, boff[l - A_LOADS], (s + st0) * kWTileElts * 2,
                        st + A_ELTS + (wave * B_LOADS + l - A_LOADS) * RPL * BK);
  };

  // 32x32x16 operands: lane (h, r) holds row r of a 32-row block, k 8h..8h+7
  // of a 16-k slice; fragments double-buffered by slice parity
  const int h = lane >> 5, r32 = lane & 31;
  bf16x8_t fa[2][Q], fb[2][Q];
  // fragment r (0..2Q-1) of slice sl, in first-use order: a0 b0 .. b(Q-1) a1 .. a(Q-1)
  auto read_frag = [&](int slot, int sl, int r) __attribute__((always_inline)) {
    const bf16_t* a = smem + slot * STAGE;
    if (r == 0)
      fa[sl & 1][0] = __builtin_bit_cast(bf16x8_t, *(const uint4*)(a + swz(wm * WT + r32, 2 * sl + h)));
    else if (r <= Q)
      fb[sl & 1][r - 1] =
          __builtin_bit_cast(bf16x8_t, *(const uint4*)(a + A_ELTS + swz(wn * WT + (r - 1) * 32 + r32, 2 * sl + h)));
    else
      fa[sl & 1][r - Q] = __builtin_bit_cast(bf16x8_t, *(const uint4*)(a + swz(wm * WT + (r - Q) * 32 + r32, 2 * sl + h)));
  };
  f32x16_t acc[Q][Q];
#pragma unroll
  for (int i = 0; i < Q; ++i)
#pragma unroll
    for (int j = 0; j < Q; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
  // an (empty) AGPR operand makes the compiler select the AGPR form of the
  // MFMAs, which keeps the accumulators in place in the AGPR file
  asm volatile("" ::"a"(0.f));
  auto mfma = [&](int sl, int q) __attribute__((always_inline)) {
    acc[q / Q][q % Q] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[sl & 1][q / Q], fb[sl & 1][q % Q], acc[q / Q][q % Q], 0, 0, 0);
  };

  // stage st; `full` = st + 2 < T (every condition below holds)
  // slotc: std::integral_constant<int, st & 1> where the caller knows the
  // parity (LDS slot addresses then fold into instruction offsets), else an
  // int and the slot is computed
  auto stage = [&](int st, bool full, auto slotc) __attribute__((always_inline)) {
    int slot;
    if constexpr (std::is_same_v<decltype(slotc), int>) slot = st & 1;
    else slot = decltype(slotc)::value;
    const bool more = full || st + 1 < T;
    const bool dma_next = st > 0 && st + 1 < T;  // rest of stage st+1 (stage 1 comes whole with the prologue)
    const bool dma_far = full || st + 2 < T;     // first part of stage st+2
    auto slice = [&](auto slc) __attribute__((always_inline)) {
      constexpr int sl = decltype(slc)::value;
      constexpr int DN = sl == 0 ? D0 : sl == 1 ? D1 : sl == 3 ? D3 : 0;
      constexpr int DB = sl == 0 ? D3 : sl == 1 ? D3 + D0 : 0;
      const int rslot = sl == 3 ? slot ^ 1 : slot;
      const bool rd = sl < 3 || more;
      const bool dd = sl == 3 ? dma_far : dma_next;
      const int ds = sl == 3 ? st + 2 : st + 1;
      static_for<0, Q * Q>([&](auto qc) __attribute__((always_inline)) {
        constexpr int q = decltype(qc)::value;
        mfma(sl, q);
        if constexpr (q < 2 * Q) {
          if (rd) read_frag(rslot, (sl + 1) & 3, q);
        }
        if constexpr (q >= DMA_AT && (q - DMA_AT) % DMA_EVERY == 0 && (q - DMA_AT) / DMA_EVERY < DN) {
          if (dd) dma(ds, sl == 3 ? slot : slot ^ 1, DB + (q - DMA_AT) / DMA_EVERY);
        }
      });
      if (full) {
        static_for<0, Q * Q>([&](auto qc) __attribute__((always_inline)) {
          constexpr int q = decltype(qc)::value;
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                    // MFMA
          if constexpr (q < 2 * Q) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // LDS read
          if constexpr (q >= DMA_AT && (q - DMA_AT) % DMA_EVERY == 0 && (q - DMA_AT) / DMA_EVERY < DN)
            __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);                  // VMEM read (DMA)
        });
      }
      if constexpr (sl == 2) {
        __builtin_amdgcn_sched_barrier(0);
        if (more) {
          wait_vmcnt_lgkm0<0>();  // stage st+1 landed, this stage's reads returned
          lds_barrier_pinned();
        }
      }
    };
    slice(std::integral_constant<int, 0>{});
    slice(std::integral_constant<int, 1>{});
    slice(std::integral_constant<int, 2>{});
    slice(std::integral_constant<int, 3>{});
  };

  // prologue: stages 0 and 1 whole, stage 0 landed everywhere, its first
  // fragments read
#pragma unroll
  for (int l = 0; l < LOADS; ++l) dma(0, 0, l);
  if (T > 1) {
#pragma unroll
    for (int l = 0; l < LOADS; ++l) dma(1, 1, l);
    wait_vmcnt_lgkm0<LOADS>();
  } else {
    wait_vmcnt_lgkm0<0>();
  }
  lds_barrier_pinned();
#pragma unroll
  for (int r = 0; r < 2 * Q; ++r) read_frag(0, 0, r);
  int st = 0;
  using S0 = std::integral_constant<int, 0>;
  using S1 = std::integral_constant<int, 1>;
  for (; st + 3 < T; st += 2) {  // two stages per trip: both slots known at compile time
    stage(st, true, S0{});
    stage(st + 1, true, S1{});
  }
  if (st + 2 < T) stage(st++, true, S0{});  // st is even here
  for (; st < T; ++st) stage(st, false, 0);

  // epilogue: acc[i][j][r] is C[32 i + 8 (r / 4) + 4 h + r % 4][32 j + r32]
  // of the wave tile. Each 32-row block goes through a wave-private LDS
  // staging area (fp32, rows padded to 136 floats: the two lane halves,
  // 4 rows apart, land 32 banks apart), then every lane reads V consecutive
  // columns and the global stores (and residual loads) are 16 bytes per
  // lane: a few wide VMEM instructions instead of one per (row group,
  // column block). SwiGLU: the wave's column blocks alternate gate and up
  // (the 32-row interleave of w_gate_up), block 2p pairs with 2p + 1.
  constexpr int ROWF = 136;
  const int rbase = m0 + wm * WT, cbase = n0 + wn * WT;
  constexpr int V = std::is_same<TC, bf16_t>::value ? 8 : 4;  // columns per lane
  constexpr int OUT_COLS = EPI == 2 ? WT / 2 : WT;
  constexpr int LPR = OUT_COLS / V, RPP = 64 / LPR;  // lanes per row, rows per pass
  const long ldc = EPI == 2 ? N / 2 : N;
  const long ccol = EPI == 2 ? cbase / 2 : cbase;
  C += (long)ks * M * ldc;  // this split's partial
  constexpr int NPASS = 32 / RPP;
  // residual operand of one pass: V values of row `row` from column `oc`
  using RRaw = typename std::conditional<std::is_same<TR, float>::value, float4,
                                         typename std::conditional<V == 8, uint4, uint2>::type>::type;
  constexpr int RCH = std::is_same<TR, float>::value ? V / 4 : 1;  // RRaw loads per pass
  // Residual loads run one 32-row block ahead of the block being stored
  // (two register sets), the first block's issued before the staging
  // barrier, so that the HBM latency of the loads, which every CU issues at
  // about the same moment, is exposed once per tile instead of once per
  // block. Block i + 1's rows are disjoint from block i's, so the loads may
  // precede block i's stores even where R aliases C, and every element is
  // still read before it is written.
  RRaw rr[2][EPI == 1 ? NPASS : 1][RCH];
  auto load_r = [&](int i) __attribute__((always_inline)) {
    if constexpr (EPI == 1) {
#pragma unroll
      for (int pass = 0; pass < NPASS; ++pass) {
        const int row = rbase + i * 32 + pass * RPP + lane / LPR, oc = (lane % LPR) * V;
        const long idx = (long)min(row, M - 1) * ldc + ccol + oc;  // rows past M: a valid row, result unused
#pragma unroll
        for (int q = 0; q < RCH; ++q) rr[i & 1][pass][q] = *(const RRaw*)(R + idx + q * 4);
      }
    }
  };
  load_r(0);
  lds_barrier_pinned();  // every wave is done reading operand slots
  float* stg = (float*)smem + wave * (32 * ROWF);
#pragma unroll
  for (int i = 0; i < Q; ++i) {
    if (i + 1 < Q) load_r(i + 1);
#pragma unroll
    for (int j = 0; j < Q; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) stg[(8 * (r >> 2) + 4 * h + (r & 3)) * ROWF + j * 32 + r32] = acc[i][j][r];
    // LDS accesses of one wave complete in order: the reads below see the writes
#pragma unroll
    for (int pass = 0; pass < NPASS; ++pass) {
      const int lr = pass * RPP + lane / LPR, oc = (lane % LPR) * V;
      const int row = rbase + i * 32 + lr;
      float v[V];
      if constexpr (EPI == 2) {
        const int p = oc / 32, c = oc % 32;
        const float* g = stg + lr * ROWF + p * 64 + c;
#pragma unroll
        for (int e = 0; e < V; e += 4) {
          const float4 gv = *(const float4*)(g + e), uv = *(const float4*)(g + 32 + e);
          v[e] = silu_fast(gv.x) * uv.x;
          v[e + 1] = silu_fast(gv.y) * uv.y;
          v[e + 2] = silu_fast(gv.z) * uv.z;
          v[e + 3] = silu_fast(gv.w) * uv.w;
        }
      } else {
#pragma unroll
        for (int e = 0; e < V; e += 4) {
          const float4 a4 = *(const float4*)(stg + lr * ROWF + oc + e);
          v[e] = a4.x;
          v[e + 1] = a4.y;
          v[e + 2] = a4.z;
          v[e + 3] = a4.w;
        }
      }
      if constexpr (EPI == 1) {
        if constexpr (std::is_same<TR, float>::value) {
#pragma unroll
          for (int q = 0; q < RCH; ++q) {
            v[4 * q] += rr[i & 1][pass][q].x;
            v[4 * q + 1] += rr[i & 1][pass][q].y;
            v[4 * q + 2] += rr[i & 1][pass][q].z;
            v[4 * q + 3] += rr[i & 1][pass][q].w;
          }
        } else if constexpr (V == 8) {
          const uint32_t w4[4] = {rr[i & 1][pass][0].x, rr[i & 1][pass][0].y, rr[i & 1][pass][0].z, rr[i & 1][pass][0].w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            v[2 * e] += bf_lo(w4[e]);
            v[2 * e + 1] += bf_hi(w4[e]);
          }
        } else {
          v[0] += bf_lo(rr[i & 1][pass][0].x);
          v[1] += bf_hi(rr[i & 1][pass][0].x);
          v[2] += bf_lo(rr[i & 1][pass][0].y);
          v[3] += bf_hi(rr[i & 1][pass][0].y);
        }
      }
      if (row >= M) continue;
      const long idx = (long)row * ldc + ccol + oc;
      if constexpr (std::is_same<TC, bf16_t>::value) {
        typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
        __builtin_nontemporal_store(u32x4{pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3]), pack_bf2(v[4], v[5]),
                                          pack_bf2(v[6], v[7])}, (u32x4*)(C + idx));
      } else {
        typedef float f32x4 __attribute__((ext_vector_type(4)));
        __builtin_nontemporal_store(f32x4{v[0], v[1], v[2], v[3]}, (f32x4*)(C + idx));
      }
    }
  }
}

// ==================================================================== skinny
// Decode-sized M (<= 64): the weight stream is the whole cost (AI = M
// FLOP/byte). A workgroup owns 64 WN weight rows (output columns) and a K
// range; its four waves own 16 WN rows each. Stages of 64 k hold the
// activation tile [16 MB rows][64] and the weight tile [64 WN rows][64];
// both are filled by global->LDS DMA into an NS-deep ring, so the bytes in
// flight cost no registers, and one barrier per stage recycles the slot.
// LDS rows are 128 B with 16-byte chunks XOR-swizzled by row % 8 (the DMA
// lane order is chosen so the fill lands swizzled). Per 32-wide k step a
// wave does MB x WN v_mfma_f32_16x16x32_bf16 with A = activations, B = W.
// With one K split the epilogue is applied from registers; otherwise fp32
// partials go to the workspace and gemm_reduce_kernel sums them in split
// order.
namespace skinny {
constexpr int NT = 256;
constexpr int KS = 64;    // k per stage
constexpr int NS = 4;     // ring depth
constexpr int MAXM = 64;
template <int MB, int WN>
constexpr size_t lds_bytes() { return (size_t)NS * (16 * MB + 64 * WN) * KS * 2; }
}  // namespace skinny

template <int MB, int WN, int EPI, typename TR, typename TC, bool DIRECT>
__global__ __launch_bounds__(256) void gemm_skinny_kernel(const bf16_t* __restrict__ A, const bf16_t* __restrict__ W,
                                                          float* __restrict__ part, const TR* __restrict__ R,
                                                          TC* __restrict__ C, int M, int N, int K, int S) {
  using namespace skinny;
  static_assert(!(DIRECT && EPI == 2) || WN == 2, "in-kernel SwiGLU pairs a gate and an up block per wave");
  static_assert(KS == kWTile, "one W tile per stage");
  constexpr int AROWS = 16 * MB, WROWS = 64 * WN;
  constexpr int STAGE = (AROWS + WROWS) * KS;  // bf16 elements
  constexpr int TA = AROWS / 8;                // A DMA instructions per stage (8 rows each), round-robin
  constexpr int WI = WROWS / 8 / 4;            // W DMA instructions per wave per stage
  extern __shared__ __attribute__((aligned(16))) bf16_t smem[];
  const int n0 = blockIdx.x * WROWS;
  const int split = blockIdx.y;
  // split `split` of S takes 64-k stages [split TT / S, (split + 1) TT / S): near-equal ranges for any S
  const int TT = K / KS;
  const int st0 = split * TT / S;
  const int T = (split + 1) * TT / S - st0;
  const int kb = st0 * KS;
  const int kps = T * KS;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4, c = lane & 15;
  // DMA lane mapping: an instruction fills 8 rows; lane l lands in row l/8 at
  // chunk l%8, which holds global chunk (l%8) ^ (row%8)
  const int drow = lane >> 3, dch = (lane & 7) ^ (lane >> 3);
  const int n_ai = (TA - wave + 3) / 4;  // this wave's A instructions (0..2)
  // DMA sources: buffer resources at the split's first activation column and
  // at the workgroup's first W tile of the split, 32-bit lane byte offsets
  const __amdgpu_buffer_rsrc_t rA = buffer_rsrc(A + kb, (uint32_t)((long)(M - 1) * K + kps) * 2);
  const __amdgpu_buffer_rsrc_t rW = buffer_rsrc(W + ((long)(n0 >> 6) * (K / 64) + kb / 64) * kWTileElts,
                                                (uint32_t)((WN - 1) * (K / 64) + kps / 64) * kWTileElts * 2);
  uint32_t aoff[2], woff[WI];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int row = (wave + 4 * i) * 8 + drow;
    aoff[i] = ((uint32_t)min(row, M - 1) * K + dch * 8) * 2;
  }
  // tiled W: the stage's 64 k of each 64-row block is one contiguous tile
#pragma unroll
  for (int i = 0; i < WI; ++i) {
    const int r = (wave * WI + i) * 8 + drow;  // row within the workgroup's WN blocks
    woff[i] = ((uint32_t)(r >> 6) * (K / 64) * kWTileElts + (r & 63) * 64 + dch * 8) * 2;
  }
  auto dma = [&](int t, int slot) {
    bf16_t* st = smem + slot * STAGE;
#pragma unroll
    for (int i = 0; i < 2; ++i)
      if (i < n_ai) load_lds16_buf(rA, aoff[i] + t * KS * 2, st + (wave + 4 * i) * 8 * KS);
#pragma unroll
    for (int i = 0; i < WI; ++i) load_lds16_buf_nt(rW, woff[i] + t * kWTileElts * 2, st + AROWS * KS + (wave * WI + i) * 8 * KS);
  };
  // this wave's own fills older than the most recent stage have landed
  auto wait_prev_stage = [&]() {
    if (n_ai == 2) wait_vmcnt_lgkm0<(NS - 2) * (WI + 2)>();
    else if (n_ai == 1) wait_vmcnt_lgkm0<(NS - 2) * (WI + 1)>();
    else wait_vmcnt_lgkm0<(NS - 2) * WI>();
  };
  auto swz = [](int row, int ch) { return row * KS + ((ch ^ (row & 7)) << 3); };
  // weight rows of n-block nb for this wave; for SwiGLU (WN 2) block 0 is a
  // gate block and block 1 the matching up block of the 32-row interleave
  auto wrow = [&](int nb) {
    if constexpr (EPI == 2 && WN == 2) {
      const int q = wave >> 1, h = wave & 1;
      return 64 * q + 32 * nb + 16 * h + c;
    } else {
      return wave * 16 * WN + nb * 16 + c;
    }
  };
  f32x4_t acc[WN][MB];
#pragma unroll
  for (int nb = 0; nb < WN; ++nb)
#pragma unroll
    for (int i = 0; i < MB; ++i) acc[nb][i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  auto compute = [&](int slot) {
    const bf16_t* st = smem + slot * STAGE;
    const bf16_t* wt = st + AROWS * KS;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      bf16x8_t wf[WN];
#pragma unroll
      for (int nb = 0; nb < WN; ++nb) wf[nb] = __builtin_bit_cast(bf16x8_t, *(const uint4*)(wt + swz(wrow(nb), 4 * j + g)));
#pragma unroll
      for (int i = 0; i < MB; ++i) {
        const bf16x8_t af = __builtin_bit_cast(bf16x8_t, *(const uint4*)(st + swz(16 * i + c, 4 * j + g)));
#pragma unroll
        for (int nb = 0; nb < WN; ++nb)
          acc[nb][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, wf[nb], acc[nb][i], 0, 0, 0);
      }
    }
  };
#pragma unroll
  for (int d = 0; d < NS - 1; ++d)
    if (d < T) dma(d, d);
  int slot = 0, fill = NS - 1, t = 0;
  // steady state: every stage refills the slot freed by the previous one
  for (; t + NS - 1 < T; ++t) {
    wait_prev_stage();
    lds_barrier();
    dma(t + NS - 1, fill);
    compute(slot);
    if (++slot == NS) slot = 0;
    if (++fill == NS) fill = 0;
  }
  for (; t < T; ++t) {  // drain
    wait_vmcnt_lgkm0<0>();
    lds_barrier();
    compute(slot);
    if (++slot == NS) slot = 0;
  }
  // acc[nb][i][r] = C[16i + 4g + r][n0 + wrow(nb)]
  if constexpr (DIRECT) {
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = 16 * i + 4 * g + r;
        if (row >= M) continue;
        if constexpr (EPI == 2) {
          const int q = wave >> 1, h = wave & 1;
          const int col = n0 / 2 + 32 * q + 16 * h + c;
          st_elt<TC>(C, (long)row * (N / 2) + col, silu_fast(acc[0][i][r]) * acc[1][i][r]);
        } else {
#pragma unroll
          for (int nb = 0; nb < WN; ++nb) {
            const long idx = (long)row * N + n0 + wrow(nb);
            float v = acc[nb][i][r];
            if constexpr (EPI == 1) v += ld_elt<TR>(R, idx);
            st_elt<TC>(C, idx, v);
          }
        }
      }
  } else {
    float* pp = part + (long)split * M * N;
#pragma unroll
    for (int nb = 0; nb < WN; ++nb)
#pragma unroll
      for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int row = 16 * i + 4 * g + r;
          if (row < M) pp[(long)row * N + n0 + wrow(nb)] = acc[nb][i][r];
        }
  }
}

// Sum split partials in split order, then apply the epilogue.
template <int EPI, typename TR, typename TC>
__global__ __launch_bounds__(256) void gemm_reduce_kernel(const float* __restrict__ part, const TR* __restrict__ R,
                                                          TC* __restrict__ C, int M, int N, int S) {
  const long total = (EPI == 2) ? (long)M * (N / 2) : (long)M * N;
  for (long e = (long)blockIdx.x * 256 + threadIdx.x; e < total; e += (long)gridDim.x * 256) {
    if constexpr (EPI == 2) {
      const int ldc = N / 2;
      const long row = e / ldc;
      const int j = (int)(e - row * ldc);
      const int gcol = (j / kGateUpBlock) * (2 * kGateUpBlock) + (j % kGateUpBlock);
      float gs = 0.f, us = 0.f;
      for (int s = 0; s < S; ++s) {
        gs += part[((long)s * M + row) * N + gcol];
        us += part[((long)s * M + row) * N + gcol + kGateUpBlock];
      }
      st_elt<TC>(C, e, silu_fast(gs) * us);
    } else {
      float v = 0.f;
      for (int s = 0; s < S; ++s) v += part[(long)s * M * N + e];
      if constexpr (EPI == 1) v += ld_elt<TR>(R, e);
      st_elt<TC>(C, e, v);
    }
  }
}

// ======================================================================= f32
template <int EPI, typename TR, typename TC>
__global__ __launch_bounds__(256) void gemm_f32_kernel(const float* __restrict__ A, const float* __restrict__ W,
                                                       const TR* __restrict__ R, TC* __restrict__ C, int M, int N,
                                                       int K) {
  __shared__ float sA[16][65], sW[16][65];
  const int m0 = blockIdx.y * 64, n0 = blockIdx.x * 64;
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += 16) {
    for (int e = threadIdx.x; e < 64 * 16; e += 256) {
      const int r = e >> 4, kk = e & 15;
      const int k = k0 + kk;
      sA[kk][r] = (m0 + r < M && k < K) ? A[(long)(m0 + r) * K + k] : 0.f;
      sW[kk][r] = (n0 + r < N && k < K) ? W[tiled_index(n0 + r, k, K)] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      float a[4], w[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        a[i] = sA[kk][ty * 4 + i];
        w[i] = sW[kk][tx * 4 + i];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], w[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = m0 + ty * 4 + i;
    if (row >= M) continue;
    if constexpr (EPI == 2) {
      continue;  // handled below through LDS
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int col = n0 + tx * 4 + j;
        if (col < N) {
          float v = acc[i][j];
          if constexpr (EPI == 1) v += ld_elt<TR>(R, (long)row * N + col);
          st_elt<TC>(C, (long)row * N + col, v);
        }
      }
    }
  }
  if constexpr (EPI == 2) {
    // SwiGLU: exchange the up half through LDS (reuse sA as [64][65])
    __shared__ float sUp[64][33];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int cl = tx * 4 + j;
        if (cl >= kGateUpBlock) sUp[ty * 4 + i][cl - kGateUpBlock] = acc[i][j];
      }
    __syncthreads();
    const int ldc = N / 2;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = m0 + ty * 4 + i;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int cl = tx * 4 + j;
        if (cl < kGateUpBlock && row < M) {
          const int col = n0 / 2 + cl;
          st_elt<TC>(C, (long)row * ldc + col, silu_f(acc[i][j]) * sUp[ty * 4 + i][cl]);
        }
      }
    }
  }
}

// ==================================================================== launch
template <int EPI, typename TR, typename TC>
static int launch_tile(int M, int N, int K, const void* A, const void* W, const void* R, void* C, hipStream_t st,
                       int splits = 1) {
  static_assert(tile::LDS_BYTES <= 160 * 1024, "LDS per workgroup");
  static const hipError_t attr = hipFuncSetAttribute((const void*)gemm_tile_kernel<EPI, TR, TC>,
                                                      hipFuncAttributeMaxDynamicSharedMemorySize, (int)tile::LDS_BYTES);
  if (attr != hipSuccess) return -1;
  const int tiles_m = (M + tile::BM - 1) / tile::BM, tiles_n = N / tile::BN;
  // wide outputs walk 8 tile-rows per group (more W reuse per XCD), narrow 4
  const int group = tiles_n >= 64 ? 8 : 4;
  hipLaunchKernelGGL((gemm_tile_kernel<EPI, TR, TC>), dim3(tiles_m * tiles_n * splits), dim3(tile::NT),
                     tile::LDS_BYTES, st, (const bf16_t*)A, (const bf16_t*)W, (const TR*)R, (TC*)C, M, N, K, tiles_n,
                     group, splits);
  return 0;
}

int compute_units() {
  static const int n = [] {
    int dev = 0, v = 0;
    if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) !=
                                                 hipSuccess || v <= 0)
      return 256;
    return v;
  }();
  return n;
}

// Cost of a tile-kernel launch of `tiles` tiles split S ways in K: rounds of
// workgroups over the compute units (one resident per unit: the kernel takes
// the whole register file) times the stages per workgroup, plus the split
// partials' traffic (written, then read once by the consumer) in stage-times:
// one 256x256x64 stage is ~1.2 us at the power-capped MFMA clock, in which
// HBM moves ~6 MB.
static double tile_cost(long tiles, int T, int S, long M, long N) {
  const long cu = compute_units();
  const long rounds = (tiles * S + cu - 1) / cu;
  return (double)rounds * ((T + S - 1) / S) + (S > 1 ? (double)S * M * N * 8.0 / 6.0e6 : 0.0);
}

int gemm_tile_splits(int M, int N, int K) {
  using namespace tile;
  if (M <= skinny::MAXM || N % BN || K % BK) return 1;
  const long tiles = (long)((M + BM - 1) / BM) * (N / BN);
  const int T = K / BK;
  int best = 1;
  double best_cost = tile_cost(tiles, T, 1, M, N);
  for (int S = 2; S <= 4 && T / S >= 16; ++S) {
    const double c = tile_cost(tiles, T, S, M, N);
    if (c < best_cost) best = S, best_cost = c;
  }
  return best;
}

size_t gemm_tile_partials_bound(int max_rows, int N, int K) {
  size_t b = 0;
  for (int m = tile::BM;; m += tile::BM) {
    const int mm = std::min(m, max_rows);
    const int S = gemm_tile_splits(mm, N, K);
    if (S > 1) b = std::max(b, (size_t)S * mm * N * sizeof(float));
    if (mm == max_rows) break;
  }
  return b;
}

int launch_gemm_tile_split(int M, int N, int K, int S, const void* A, const void* W, float* part, hipStream_t st) {
  if (M <= 0 || S < 1 || N % tile::BN || K % tile::BK || K / tile::BK < S) return -1;
  return launch_tile<0, float, float>(M, N, K, A, W, nullptr, part, st, S);
}

template <int EPI, typename TR, typename TC>
static int launch_reduce(int M, int N, int S, const float* part, const void* R, void* C, hipStream_t st);

int launch_split_residual(int r_dt, int c_dt, int M, int N, int S, const float* part, const void* R, void* C,
                          hipStream_t st) {
  if (M == 0) return 0;
  if (r_dt == 0 && c_dt == 1) return launch_reduce<1, float, bf16_t>(M, N, S, part, R, C, st);
  if (r_dt == 1 && c_dt == 1) return launch_reduce<1, bf16_t, bf16_t>(M, N, S, part, R, C, st);
  if (r_dt == 1 && c_dt == 0) return launch_reduce<1, bf16_t, float>(M, N, S, part, R, C, st);
  if (r_dt == 0 && c_dt == 0) return launch_reduce<1, float, float>(M, N, S, part, R, C, st);
  return -1;
}

template <typename TR, typename TC>
__global__ __launch_bounds__(256) void gemm_reduce_residual4_kernel(const float* __restrict__ part,
                                                                    const TR* __restrict__ R, TC* __restrict__ C,
                                                                    long n4, long mn, int S) {
  for (long e = (long)blockIdx.x * 256 + threadIdx.x; e < n4; e += (long)gridDim.x * 256) {
    float4 v = ((const float4*)part)[e];
    for (int s = 1; s < S; ++s) {
      const float4 p = ((const float4*)(part + s * mn))[e];
      v.x += p.x, v.y += p.y, v.z += p.z, v.w += p.w;
    }
    if constexpr (std::is_same<TR, float>::value) {
      const float4 r = ((const float4*)R)[e];
      v.x += r.x, v.y += r.y, v.z += r.z, v.w += r.w;
    } else {
      const uint2 r = ((const uint2*)R)[e];
      v.x += __uint_as_float(r.x << 16), v.y += __uint_as_float(r.x & 0xffff0000u);
      v.z += __uint_as_float(r.y << 16), v.w += __uint_as_float(r.y & 0xffff0000u);
    }
    if constexpr (std::is_same<TC, float>::value)
      ((float4*)C)[e] = v;
    else
      ((uint2*)C)[e] = uint2{pack_bf2(v.x, v.y), pack_bf2(v.z, v.w)};
  }
}

template <int EPI, typename TR, typename TC>
static int launch_reduce(int M, int N, int S, const float* part, const void* R, void* C, hipStream_t st) {
  const long total = (EPI == 2) ? (long)M * (N / 2) : (long)M * N;
  if constexpr (EPI == 1) {
    auto al = [](const void* p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; };
    if (N % 4 == 0 && al(part, 16) && al(R, 4 * sizeof(TR)) && al(C, 4 * sizeof(TC))) {
      const long n4 = total / 4;
      const int blocks = (int)std::min<long>((n4 + 255) / 256, 8192);
      hipLaunchKernelGGL((gemm_reduce_residual4_kernel<TR, TC>), dim3(blocks), dim3(256), 0, st, part, (const TR*)R,
                         (TC*)C, n4, total, S);
      return 0;
    }
  }
  int blocks = (int)std::min<long>((total + 255) / 256, 4096);
  hipLaunchKernelGGL((gemm_reduce_kernel<EPI, TR, TC>), dim3(blocks), dim3(256), 0, st, part, (const TR*)R, (TC*)C,
                     M, N, S);
  return 0;
}

// Skinny launch plan: WN 64-row blocks per workgroup and S K-splits. Two
// blocks per workgroup halve the activation traffic per weight byte and win
// whenever the grid still reaches ~160 workgroups; otherwise one block. The
// split count is the largest that keeps the grid within one round of 256
// workgroups, at most 8, while each split keeps at least 16 stages (shorter
// splits lose more to ring fill and drain than they gain in parallelism, and
// add partial-sum traffic); splits are near-equal stage ranges, so any count
// works. Chosen from a sweep of both widths and 1..8 splits over the 8B and
// 70B decode shapes at M = 32 and 64, reduction included.
static int skinny_splits_for(int tiles, int K, int target) {
  using namespace skinny;
  const int stages = K / KS;
  int S = std::max(1, std::min(8, target / tiles));
  while (S > 1 && stages / S < 16) --S;
  return S;
}

SkinnyPlan gemm_skinny_plan(int M, int N, int K) {
  (void)M;
  if (N % 128 == 0) {
    const int S = skinny_splits_for(N / 128, K, 256);
    if ((N / 128) * S >= 160) return {2, S};
  }
  return {1, skinny_splits_for(N / 64, K, 256)};
}

template <int MB, int WN, int EPI, typename TR, typename TC, bool DIRECT>
static int launch_skinny_k(int M, int N, int K, int S, const void* A, const void* W, float* part, const void* R,
                           void* C, hipStream_t st) {
  constexpr size_t lds = skinny::lds_bytes<MB, WN>();
  static const hipError_t attr = hipFuncSetAttribute(
      (const void*)gemm_skinny_kernel<MB, WN, EPI, TR, TC, DIRECT>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (attr != hipSuccess) return -1;
  hipLaunchKernelGGL((gemm_skinny_kernel<MB, WN, EPI, TR, TC, DIRECT>), dim3(N / (64 * WN), S), dim3(skinny::NT), lds,
                     st, (const bf16_t*)A, (const bf16_t*)W, part, (const TR*)R, (TC*)C, M, N, K, S);
  return 0;
}

template <int MB, int WN, int EPI, typename TR, typename TC>
static int launch_skinny_wn(int M, int N, int K, int S, const void* A, const void* W, float* part, const void* R,
                            void* C, hipStream_t st) {
  if constexpr (EPI != 2 || WN == 2) {
    if (S == 1) return launch_skinny_k<MB, WN, EPI, TR, TC, true>(M, N, K, 1, A, W, part, R, C, st);
  }
  if (launch_skinny_k<MB, WN, EPI, TR, TC, false>(M, N, K, S, A, W, part, R, C, st)) return -1;
  return launch_reduce<EPI, TR, TC>(M, N, S, part, R, C, st);
}

template <int MB, int EPI, typename TR, typename TC>
static int launch_skinny_mb(int M, int N, int K, SkinnyPlan pl, const void* A, const void* W, float* part,
                            const void* R, void* C, hipStream_t st) {
  if (pl.wn == 2) return launch_skinny_wn<MB, 2, EPI, TR, TC>(M, N, K, pl.s, A, W, part, R, C, st);
  return launch_skinny_wn<MB, 1, EPI, TR, TC>(M, N, K, pl.s, A, W, part, R, C, st);
}

template <int EPI, typename TR, typename TC>
static int launch_skinny_plan(int M, int N, int K, SkinnyPlan pl, const void* A, const void* W, float* part,
                              const void* R, void* C, hipStream_t st) {
  if ((pl.wn != 1 && pl.wn != 2) || N % (64 * pl.wn) != 0 || pl.s < 1 || K / skinny::KS < pl.s) return -1;
  switch ((M + 15) / 16) {
    case 1: return launch_skinny_mb<1, EPI, TR, TC>(M, N, K, pl, A, W, part, R, C, st);
    case 2: return launch_skinny_mb<2, EPI, TR, TC>(M, N, K, pl, A, W, part, R, C, st);
    case 3: return launch_skinny_mb<3, EPI, TR, TC>(M, N, K, pl, A, W, part, R, C, st);
    case 4: return launch_skinny_mb<4, EPI, TR, TC>(M, N, K, pl, A, W, part, R, C, st);
    default: return -1;
  }
}

template <int EPI, typename TR, typename TC>
static int launch_skinny(int M, int N, int K, const void* A, const void* W, float* part, const void* R, void* C,
                         hipStream_t st) {
  return launch_skinny_plan<EPI, TR, TC>(M, N, K, gemm_skinny_plan(M, N, K), A, W, part, R, C, st);
}

template <int EPI, typename TR, typename TC>
static int launch_f32(int M, int N, int K, const void* A, const void* W, const void* R, void* C, hipStream_t st) {
  dim3 grid((N + 63) / 64, (M + 63) / 64);
  hipLaunchKernelGGL((gemm_f32_kernel<EPI, TR, TC>), grid, dim3(256), 0, st, (const float*)A, (const float*)W,
                     (const TR*)R, (TC*)C, M, N, K);
  return 0;
}

size_t gemm_workspace_bytes(int dtype, int M, int N, int K) {
  if (dtype != 1 || M > skinny::MAXM) return 0;
  return (size_t)gemm_skinny_plan(M, N, K).s * M * N * sizeof(float);
}

// Dispatch on (dtype, r_dtype, c_dtype, epilogue) and on M.
int launch_gemm(int dtype, int r_dt, int c_dt, int epi, int M, int N, int K, const void* A, const void* W,
                const void* R, void* C, void* ws, size_t ws_bytes, hipStream_t st) {
  if (M == 0) return 0;
  if (dtype == 0) {
    if (N % 64 != 0 && epi == 2) return -1;
#define F32_CASE(E, TR_, TC_, rd, cd) \
  if (epi == E && r_dt == rd && c_dt == cd) return launch_f32<E, TR_, TC_>(M, N, K, A, W, R, C, st);
    F32_CASE(0, float, float, 0, 0)
    F32_CASE(0, float, float, 1, 0)
    F32_CASE(1, float, float, 0, 0)
    F32_CASE(2, float, float, 0, 0)
    F32_CASE(2, float, float, 1, 0)
#undef F32_CASE
    return -1;
  }
  if (K % 64 != 0) return -1;
  if (M <= skinny::MAXM && N % 64 == 0) {
    if (ws_bytes < gemm_workspace_bytes(dtype, M, N, K)) return -2;
    float* part = (float*)ws;
#define SK_CASE(E, TR_, TC_, rd, cd) \
  if (epi == E && r_dt == rd && c_dt == cd) return launch_skinny<E, TR_, TC_>(M, N, K, A, W, part, R, C, st);
    SK_CASE(0, float, bf16_t, 0, 1)
    SK_CASE(0, float, bf16_t, 1, 1)
    SK_CASE(0, float, float, 0, 0)
    SK_CASE(0, float, float, 1, 0)
    SK_CASE(1, bf16_t, float, 1, 0)
    SK_CASE(1, float, bf16_t, 0, 1)
    SK_CASE(1, bf16_t, bf16_t, 1, 1)
    SK_CASE(1, float, float, 0, 0)
    SK_CASE(2, float, bf16_t, 0, 1)
    SK_CASE(2, float, bf16_t, 1, 1)
    SK_CASE(2, float, float, 0, 0)
#undef SK_CASE
    return -1;
  }
  if (N % 256 != 0) return -1;
#define TILE_CASE(E, TR_, TC_, rd, cd) \
  if (epi == E && r_dt == rd && c_dt == cd) return launch_tile<E, TR_, TC_>(M, N, K, A, W, R, C, st);
  TILE_CASE(0, float, bf16_t, 0, 1)
  TILE_CASE(0, float, bf16_t, 1, 1)
  TILE_CASE(0, float, float, 0, 0)
  TILE_CASE(0, float, float, 1, 0)
  TILE_CASE(1, bf16_t, float, 1, 0)
  TILE_CASE(1, float, bf16_t, 0, 1)
  TILE_CASE(1, bf16_t, bf16_t, 1, 1)
  TILE_CASE(1, float, float, 0, 0)
  TILE_CASE(2, float, bf16_t, 0, 1)
  TILE_CASE(2, float, bf16_t, 1, 1)
  TILE_CASE(2, float, float, 0, 0)
#undef TILE_CASE
  return -1;
}

// launch_gemm, except that a decode-sized bf16 GEMM whose plan splits K in
// 2, 3, 4 or 8 stops at the split partials (fp32 [S][M][N] at the head of ws,
// summed in split order by the consumer, which fuses the reduction with its
// own work); *splits = S then, else 1 and C holds the result.
int launch_gemm_split(int dtype, int r_dt, int c_dt, int epi, int M, int N, int K, const void* A, const void* W,
                      const void* R, void* C, void* ws, size_t ws_bytes, hipStream_t st, int* splits) {
  *splits = 1;
  if (dtype == 1 && M > 0 && M <= skinny::MAXM && N % 64 == 0 && K % 64 == 0 && epi != 2) {
    const SkinnyPlan pl = gemm_skinny_plan(M, N, K);
    if (pl.s == 2 || pl.s == 3 || pl.s == 4 || pl.s == 8) {  // the split counts the fused consumers take
      if (ws_bytes < gemm_workspace_bytes(dtype, M, N, K)) return -2;
      *splits = pl.s;
      float* part = (float*)ws;
      // the partial kernel's output does not depend on the epilogue or the
      // output types (only its weight-row mapping does, for SwiGLU)
      auto go = [&](auto mbc) {
        constexpr int MB = decltype(mbc)::value;
        if (pl.wn == 2) return launch_skinny_k<MB, 2, 0, float, float, false>(M, N, K, pl.s, A, W, part, R, C, st);
        return launch_skinny_k<MB, 1, 0, float, float, false>(M, N, K, pl.s, A, W, part, R, C, st);
      };
      switch ((M + 15) / 16) {
        case 1: return go(std::integral_constant<int, 1>{});
        case 2: return go(std::integral_constant<int, 2>{});
        case 3: return go(std::integral_constant<int, 3>{});
        default: return go(std::integral_constant<int, 4>{});
      }
    }
  }
  return launch_gemm(dtype, r_dt, c_dt, epi, M, N, K, A, W, R, C, ws, ws_bytes, st);
}

// Bytes of split-K partials a bf16 launch actually writes: 0 for the tile
// path and for skinny launches that apply their epilogue in the kernel.
size_t gemm_partials_bytes(int dtype, int epi, int M, int N, int K) {
  if (dtype != 1 || M <= 0 || M > skinny::MAXM || N % 64 != 0 || K % 64 != 0) return 0;
  const SkinnyPlan pl = gemm_skinny_plan(M, N, K);
  if (pl.s == 1 && (epi != 2 || pl.wn == 2)) return 0;
  return (size_t)pl.s * M * N * sizeof(float);
}

// ------------------------------------------------------------ static scratch
// Split-K partials for callers that cannot allocate device memory: a
// file-scope device array, one copy on every GPU the library runs on, kept
// until the process ends. In host code `scratch` names a host-side stand-in,
// not a device address, so host code never passes it to a kernel or a copy:
// gemm_static_scratch() returns the device address of the current GPU's
// copy, looked up once per device with hipGetSymbolAddress.
static __device__ __align__(256) uint8_t scratch[kGemmStaticScratchBytes];

namespace {
constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxScratchDevices] = {};
}  // namespace

hipError_t gemm_static_scratch(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxScratchDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace ps

namespace ps {
// Host-side mirror of launch_gemm's dispatch conditions: 0 if supported.
int gemm_check(int dtype, int epi, int M, int N, int K) {
  if (M < 0 || N <= 0 || K <= 0) return -1;
  if (epi == 2 && N % (2 * kGateUpBlock) != 0) return -1;
  if (dtype == 0) return 0;
  if (dtype != 1 || K % 64 != 0 || K >= (1 << 21)) return -1;  // 32-bit byte offsets per 256-row tile
  if (M <= skinny::MAXM && N % 64 == 0) return 0;
  return (N % 256 == 0) ? 0 : -1;
}
}  // namespace ps
