// GEMMs of the layer: C = epilogue(A W^T), A [M, K] row-major, W [N, K]
// (the nn.Linear orientation) stored in 64x64 tiles: tile (i, j) covers rows
// 64i.. and columns 64j.., sits at tile index i * ceil(K/64) + j, and is
// row-major inside (64 rows of 64 elements). Every 64-row by 64-k slab a
// workgroup streams is then one contiguous 8 KiB (bf16) block of HBM rather
// than 64 strided 128-byte pieces. fp32 accumulation (gfx950).
//
//  * gemm_tile_kernel: prefill-sized M. 256x256x64 workgroup tile, eight
//    waves of 128x64 (two per SIMD), v_mfma_f32_16x16x32_bf16, operands
//    staged through double-buffered, XOR-swizzled LDS (128 KiB) by direct
//    global->LDS loads. MFMA-bound.
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

#include <type_traits>

namespace ps {

__device__ __forceinline__ float silu_f(float x) { return x / (1.f + expf(-x)); }

template <typename T> __device__ __forceinline__ float ld_elt(const T* p, long i);
template <> __device__ __forceinline__ float ld_elt<float>(const float* p, long i) { return p[i]; }
template <> __device__ __forceinline__ float ld_elt<bf16_t>(const bf16_t* p, long i) { return bf2f(p[i]); }
template <typename T> __device__ __forceinline__ void st_elt(T* p, long i, float v);
template <> __device__ __forceinline__ void st_elt<float>(float* p, long i, float v) { p[i] = v; }
template <> __device__ __forceinline__ void st_elt<bf16_t>(bf16_t* p, long i, float v) { p[i] = f2bf(v); }

// ====================================================================== tile
// Workgroup tile BM x BN, K step BK, WAVES_M x WAVES_N waves, STAGES-deep
// ring of LDS buffers filled by direct global->LDS loads
// (global_load_lds_dwordx4): one wave instruction fills 1 KiB of LDS, lane l
// landing at +16 l. LDS rows hold BK bf16 (BK/8 16-byte chunks), XOR-
// swizzled so that the 16-byte operand reads of 16 consecutive rows hit 16
// distinct 16-byte bank groups; the global address of each lane is chosen
// so that the linear fill lands in swizzled order.
template <int BM_, int BN_, int BK_, int WAVES_M_, int WAVES_N_, int STAGES_>
struct TileCfg {
  static constexpr int BM = BM_, BN = BN_, BK = BK_, STAGES = STAGES_;
  static constexpr int WAVES_M = WAVES_M_, WAVES_N = WAVES_N_;
  static constexpr int NW = WAVES_M * WAVES_N;
  static constexpr int NT = 64 * NW;
  static constexpr int WTM = BM / WAVES_M, WTN = BN / WAVES_N;
  static constexpr int FM = WTM / 16, FN = WTN / 16;  // 16x16 MFMA blocks per wave
  static constexpr int CPR = BK / 8;               // 16-byte chunks per LDS row
  static constexpr int ROWS_PER_LOAD = 64 / CPR;   // rows one wave instruction fills
  static constexpr int A_ELTS = BM * BK, B_ELTS = BN * BK;
  static constexpr int STAGE_ELTS = A_ELTS + B_ELTS;
  static constexpr int A_LOADS = BM / ROWS_PER_LOAD / NW;  // per wave per stage
  static constexpr int B_LOADS = BN / ROWS_PER_LOAD / NW;
  static constexpr int LOADS = A_LOADS + B_LOADS;
  static constexpr size_t LDS_BYTES = (size_t)STAGES * STAGE_ELTS * 2;
  static_assert(FM >= 1 && FN >= 1 && A_LOADS >= 1 && B_LOADS >= 1, "tile shape");
  static_assert(BM % (ROWS_PER_LOAD * NW) == 0 && BN % (ROWS_PER_LOAD * NW) == 0, "load split");
  __device__ static int swz(int row, int ch) {
    return row * BK + ((ch ^ ((row / (16 / CPR)) % CPR)) << 3);
  }
};

// One 16-byte global->LDS fill per lane (global_load_lds_dwordx4). Kept in
// a non-template device function: used directly inside a kernel template
// the builtin makes the host pass drop the kernel's instantiation.
__device__ __forceinline__ void load_lds16(const bf16_t* g, bf16_t* lds) {
  __builtin_amdgcn_global_load_lds(g, (__attribute__((address_space(3))) void*)lds, 16, 0, 0);
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

// bf16 store and SwiGLU epilogues stage the output tile in LDS
template <int EPI, typename TC>
constexpr bool staged_epilogue() { return EPI != 1 && std::is_same<TC, bf16_t>::value; }
template <class CF, int EPI>
constexpr int tile_out_stride() { return (EPI == 2 ? CF::BN / 2 : CF::BN) * 2 + 16; }
template <class CF>
constexpr int tile_res_stride() { return CF::BN * 4 + 16; }
template <class CF, int EPI, typename TC>
constexpr size_t tile_lds_bytes() {
  const size_t staged = staged_epilogue<EPI, TC>() ? (size_t)CF::BM * tile_out_stride<CF, EPI>()
                        : EPI == 1                ? (size_t)(CF::BM / 2) * tile_res_stride<CF>()
                                                  : 0;
  return CF::LDS_BYTES > staged ? CF::LDS_BYTES : staged;
}

template <class CF, int EPI, typename TR, typename TC>
__global__ __launch_bounds__(CF::NT) void gemm_tile_kernel(
    const bf16_t* __restrict__ A, const bf16_t* __restrict__ W, const TR* __restrict__ R, TC* __restrict__ C,
    int M, int N, int K, int tiles_n) {
  constexpr int BM = CF::BM, BN = CF::BN, BK = CF::BK, STAGES = CF::STAGES;
  extern __shared__ __attribute__((aligned(16))) bf16_t smem[];

  // XCD-aware tile order: consecutive workgroup ids go round-robin over the
  // 8 XCDs; give each XCD a contiguous range of tiles so that tiles sharing
  // A rows and W rows meet in the same L2.
  const int nwg = gridDim.x;
  int id = blockIdx.x;
  if ((nwg & 7) == 0) id = (id & 7) * (nwg >> 3) + (id >> 3);
  // within that order, walk groups of 4 tile-rows across N
  constexpr int GROUP = 4;
  const int tiles_m = nwg / tiles_n;
  const int group_sz = GROUP * tiles_n;
  const int grp = id / group_sz;
  const int first_m = grp * GROUP;
  const int gm = min(GROUP, tiles_m - first_m);
  const int tm = first_m + (id % group_sz) % gm;
  const int tn = (id % group_sz) / gm;
  const int m0 = tm * BM, n0 = tn * BN;

  const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
  const int wm = wave / CF::WAVES_N, wn = wave % CF::WAVES_N;
  const int g = lane >> 4, c = lane & 15;  // 16x16x32 operand / result lane roles

  // per-lane global sources of this wave's loads (row block of the wave)
  const int lrow = lane / CF::CPR, lpos = lane % CF::CPR;
  const bf16_t* ga[CF::A_LOADS];
  const bf16_t* gb[CF::B_LOADS];
#pragma unroll
  for (int i = 0; i < CF::A_LOADS; ++i) {
    const int row = (wave * CF::A_LOADS + i) * CF::ROWS_PER_LOAD + lrow;
    const int ch = lpos ^ ((row / (16 / CF::CPR)) % CF::CPR);
    ga[i] = A + (long)min(m0 + row, M - 1) * K + ch * 8;
  }
#pragma unroll
  for (int i = 0; i < CF::B_LOADS; ++i) {
    const int row = (wave * CF::B_LOADS + i) * CF::ROWS_PER_LOAD + lrow;
    const int ch = lpos ^ ((row / (16 / CF::CPR)) % CF::CPR);
    const int n = n0 + row;  // tiled W: k-tile kt of row n at ((n/64) K/64 + kt) 4096 + (n%64) 64
    gb[i] = W + (long)(n >> 6) * (K / 64) * kWTileElts + (n & 63) * 64 + ch * 8;
  }
  static_assert(BK == 64, "one W tile per k step");
  auto gload = [&](int kt, int stage) {
    bf16_t* a = smem + stage * CF::STAGE_ELTS;
    bf16_t* b = a + CF::A_ELTS;
#pragma unroll
    for (int i = 0; i < CF::A_LOADS; ++i)
      load_lds16(ga[i] + kt * BK, a + (wave * CF::A_LOADS + i) * CF::ROWS_PER_LOAD * BK);
#pragma unroll
    for (int i = 0; i < CF::B_LOADS; ++i)
      load_lds16(gb[i] + (long)kt * kWTileElts, b + (wave * CF::B_LOADS + i) * CF::ROWS_PER_LOAD * BK);
  };

  // operand fragments, double-buffered in registers across 32-wide k steps:
  // lane (g, c) holds row c of a 16-row block, k = 8 g .. 8 g + 7 of the step
  constexpr int FM = CF::FM, FN = CF::FN, KK = BK / 32;
  static_assert(KK % 2 == 0, "register double-buffering alternates buffers by k-step parity");
  bf16x8_t fa[2][FM], fb[2][FN];
  auto frags = [&](int slot, int kk, int p) {
    const bf16_t* a = smem + slot * CF::STAGE_ELTS;
    const bf16_t* b = a + CF::A_ELTS;
#pragma unroll
    for (int i = 0; i < FM; ++i)
      fa[p][i] = __builtin_bit_cast(bf16x8_t, *(const uint4*)(a + CF::swz(wm * CF::WTM + i * 16 + c, 4 * kk + g)));
#pragma unroll
    for (int j = 0; j < FN; ++j)
      fb[p][j] = __builtin_bit_cast(bf16x8_t, *(const uint4*)(b + CF::swz(wn * CF::WTN + j * 16 + c, 4 * kk + g)));
  };
  f32x4_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  auto mfmas = [&](int p) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[p][i], fb[p][j], acc[i][j], 0, 0, 0);
  };
  // issue order for one k step: the next step's LDS reads spread evenly
  // between this step's MFMAs, so read latency hides under matrix work
  auto interleave = [&]() {
    constexpr int RATIO = (FM * FN) / (FM + FN) > 0 ? (FM * FN) / (FM + FN) : 1;
#pragma unroll
    for (int q = 0; q < FM + FN; ++q) {
      __builtin_amdgcn_sched_group_barrier(0x008, RATIO, 0);  // MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);      // LDS read
    }
    if constexpr (FM * FN > RATIO * (FM + FN))
      __builtin_amdgcn_sched_group_barrier(0x008, FM * FN - RATIO * (FM + FN), 0);
  };

  const int KT = K / BK;
  // prologue: stages 0 .. STAGES-2 in flight; stage 0 landed everywhere;
  // stage STAGES-1 issued; fragments of (stage 0, k step 0) requested
#pragma unroll
  for (int st = 0; st < STAGES - 1; ++st)
    if (st < KT) gload(st, st);
  if (STAGES - 2 < KT) wait_vmcnt_lgkm0<(STAGES - 2) * CF::LOADS>();
  else wait_vmcnt_lgkm0<0>();
  lds_barrier();
  if (STAGES - 1 < KT) gload(STAGES - 1, STAGES - 1);
  frags(0, 0, 0);
  for (int kt = 0; kt < KT; ++kt) {
    const int slot = kt % STAGES;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      const int p = kk & 1;
      if (kk < KK - 1) {
        frags(slot, kk + 1, p ^ 1);
        mfmas(p);
        interleave();
      } else {
        mfmas(p);
        if (kt + 1 < KT) {
          // stage kt+1 has landed for this wave and this wave's reads of
          // stage kt have returned; after the barrier both hold for all
          // waves, so slot kt may be refilled with stage kt+STAGES
          if (kt + STAGES - 1 < KT) wait_vmcnt_lgkm0<(STAGES - 2) * CF::LOADS>();
          else wait_vmcnt_lgkm0<0>();
          lds_barrier();
          if (kt + STAGES < KT) gload(kt + STAGES, slot);
          frags((kt + 1) % STAGES, 0, p ^ 1);
        }
      }
    }
  }

  // epilogue: acc[i][j][r] = C[row 16 i + 4 g + r][col 16 j + c] of the wave tile.
  // SwiGLU pairs: the wave's columns hold 32-row gate/up blocks alternately,
  // so gate n-block jg = 4 (jp / 2) + jp % 2 pairs with up n-block jg + 2.
  const int rbase = m0 + wm * CF::WTM, cbase = n0 + wn * CF::WTN;
  auto gate_nb = [](int jp) { return 4 * (jp >> 1) + (jp & 1); };
  auto gate_col = [](int jp) { return 32 * (jp >> 1) + 16 * (jp & 1); };  // wave-local output column
  if constexpr (staged_epilogue<EPI, TC>()) {
    // bf16 results go through LDS (free after the main loop) so that global
    // stores are whole 16-byte chunks of full rows rather than 2-byte
    // scatters; padded rows put the four lane groups (rows 4 apart) on
    // different banks
    constexpr int OCOLS = EPI == 2 ? BN / 2 : BN;
    constexpr int OSTRIDE = tile_out_stride<CF, EPI>();  // bytes per staged row
    char* so = (char*)smem;
    __syncthreads();  // every wave is done reading operand tiles
#pragma unroll
    for (int i = 0; i < CF::FM; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int lrow = wm * CF::WTM + i * 16 + 4 * g + r;
        if constexpr (EPI == 2) {
#pragma unroll
          for (int jp = 0; jp < CF::FN / 2; ++jp) {
            const int lcol = (wn * CF::WTN >> 1) + gate_col(jp) + c;
            const int jg = gate_nb(jp);
            *(bf16_t*)(so + lrow * OSTRIDE + lcol * 2) = f2bf(silu_f(acc[i][jg][r]) * acc[i][jg + 2][r]);
          }
        } else {
#pragma unroll
          for (int j = 0; j < CF::FN; ++j) {
            const int lcol = wn * CF::WTN + j * 16 + c;
            *(bf16_t*)(so + lrow * OSTRIDE + lcol * 2) = f2bf(acc[i][j][r]);
          }
        }
      }
    __syncthreads();
    constexpr int CHUNKS = OCOLS / 8;  // 16-byte chunks per row
    const long ldc = EPI == 2 ? N / 2 : N;
    const int ocol0 = EPI == 2 ? n0 / 2 : n0;
    for (int q = t; q < BM * CHUNKS; q += CF::NT) {
      const int lrow = q / CHUNKS, ch = q - lrow * CHUNKS;
      if (m0 + lrow < M)
        *(uint4*)(C + (long)(m0 + lrow) * ldc + ocol0 + ch * 8) = *(const uint4*)(so + lrow * OSTRIDE + ch * 16);
    }
  } else if constexpr (EPI == 1) {
    // residual: the fp32 tile goes through LDS in two halves of 128 rows
    // (the waves with wm == half write theirs), then every thread adds R and
    // stores 4 consecutive columns per access; rows of 1040 B put the four
    // lane groups (rows 4 apart) on different banks
    static_assert(CF::WAVES_M == 2 && CF::WTM * 2 == BM, "two row halves of the tile");
    constexpr int HROWS = BM / 2;
    constexpr int FSTRIDE = tile_res_stride<CF>();  // bytes per staged row
    char* so = (char*)smem;
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      __syncthreads();  // operand tiles (first half) or the previous half are no longer read
      if (wm == half) {
#pragma unroll
        for (int i = 0; i < CF::FM; ++i)
#pragma unroll
          for (int j = 0; j < CF::FN; ++j)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const int lrow = i * 16 + 4 * g + r;
              const int lcol = wn * CF::WTN + j * 16 + c;
              *(float*)(so + lrow * FSTRIDE + lcol * 4) = acc[i][j][r];
            }
      }
      __syncthreads();
      constexpr int CHUNKS = BN / 4;  // 4 columns per access
      for (int q = t; q < HROWS * CHUNKS; q += CF::NT) {
        const int lrow = q / CHUNKS, ch = q - lrow * CHUNKS;
        const int row = m0 + half * HROWS + lrow;
        if (row >= M) continue;
        const float4 v = *(const float4*)(so + lrow * FSTRIDE + ch * 16);
        const long idx = (long)row * N + n0 + ch * 4;
        float o[4] = {v.x, v.y, v.z, v.w};
        if constexpr (std::is_same<TR, float>::value) {
          const float4 rr = *(const float4*)(R + idx);
          o[0] += rr.x; o[1] += rr.y; o[2] += rr.z; o[3] += rr.w;
        } else {
          const uint2 rr = *(const uint2*)(R + idx);
          o[0] += bf_lo(rr.x); o[1] += bf_hi(rr.x); o[2] += bf_lo(rr.y); o[3] += bf_hi(rr.y);
        }
        if constexpr (std::is_same<TC, float>::value) {
          *(float4*)(C + idx) = make_float4(o[0], o[1], o[2], o[3]);
        } else {
          *(uint2*)(C + idx) = make_uint2(pack_bf2(o[0], o[1]), pack_bf2(o[2], o[3]));
        }
      }
    }
  } else if constexpr (EPI == 2) {
    const int ldc = N / 2;
#pragma unroll
    for (int i = 0; i < CF::FM; ++i)
#pragma unroll
      for (int jp = 0; jp < CF::FN / 2; ++jp)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int row = rbase + i * 16 + 4 * g + r;
          if (row < M) {
            const int jg = gate_nb(jp);
            const int col = (cbase >> 1) + gate_col(jp) + c;
            st_elt<TC>(C, (long)row * ldc + col, silu_f(acc[i][jg][r]) * acc[i][jg + 2][r]);
          }
        }
  } else {
#pragma unroll
    for (int i = 0; i < CF::FM; ++i)
#pragma unroll
      for (int j = 0; j < CF::FN; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int row = rbase + i * 16 + 4 * g + r;
          if (row < M) st_elt<TC>(C, (long)row * N + cbase + j * 16 + c, acc[i][j][r]);
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
                                                          TC* __restrict__ C, int M, int N, int K, int kps) {
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
  const int kb = split * kps;
  const int T = kps / KS;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4, c = lane & 15;
  // DMA lane mapping: an instruction fills 8 rows; lane l lands in row l/8 at
  // chunk l%8, which holds global chunk (l%8) ^ (row%8)
  const int drow = lane >> 3, dch = (lane & 7) ^ (lane >> 3);
  const int n_ai = (TA - wave + 3) / 4;  // this wave's A instructions (0..2)
  const bf16_t* asrc[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int row = (wave + 4 * i) * 8 + drow;
    asrc[i] = A + (long)min(row, M - 1) * K + kb + dch * 8;
  }
  // tiled W: the stage's 64 k of each 64-row block is one contiguous tile
  const bf16_t* wsrc[WI];
#pragma unroll
  for (int i = 0; i < WI; ++i) {
    const int n = n0 + (wave * WI + i) * 8 + drow;
    wsrc[i] = W + ((long)(n >> 6) * (K / 64) + kb / 64) * kWTileElts + (n & 63) * 64 + dch * 8;
  }
  auto dma = [&](int t, int slot) {
    bf16_t* st = smem + slot * STAGE;
#pragma unroll
    for (int i = 0; i < 2; ++i)
      if (i < n_ai) load_lds16(asrc[i] + t * KS, st + (wave + 4 * i) * 8 * KS);
#pragma unroll
    for (int i = 0; i < WI; ++i) load_lds16(wsrc[i] + (long)t * kWTileElts, st + AROWS * KS + (wave * WI + i) * 8 * KS);
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
          st_elt<TC>(C, (long)row * (N / 2) + col, silu_f(acc[0][i][r]) * acc[1][i][r]);
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
      st_elt<TC>(C, e, silu_f(gs) * us);
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
// Default prefill tile configuration.
using TileDefault = TileCfg<256, 256, 64, 2, 4, 2>;  // 8 waves of 128x64, 2 per SIMD

template <class CF, int EPI, typename TR, typename TC>
int launch_tile_cfg(int M, int N, int K, const void* A, const void* W, const void* R, void* C, hipStream_t st) {
  constexpr int BM = CF::BM, BN = CF::BN;
  const int tiles_m = (M + BM - 1) / BM, tiles_n = N / BN;
  constexpr size_t lds = tile_lds_bytes<CF, EPI, TC>();
  static_assert(lds <= 160 * 1024, "LDS per workgroup");
  static const hipError_t attr = hipFuncSetAttribute((const void*)gemm_tile_kernel<CF, EPI, TR, TC>,
                                                      hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (attr != hipSuccess) return -1;
  hipLaunchKernelGGL((gemm_tile_kernel<CF, EPI, TR, TC>), dim3(tiles_m * tiles_n), dim3(CF::NT), lds, st,
                     (const bf16_t*)A, (const bf16_t*)W, (const TR*)R, (TC*)C, M, N, K, tiles_n);
  return 0;
}

template <int EPI, typename TR, typename TC>
static int launch_tile(int M, int N, int K, const void* A, const void* W, const void* R, void* C, hipStream_t st) {
  return launch_tile_cfg<TileDefault, EPI, TR, TC>(M, N, K, A, W, R, C, st);
}

template <int EPI, typename TR, typename TC>
static int launch_reduce(int M, int N, int S, const float* part, const void* R, void* C, hipStream_t st) {
  const long total = (EPI == 2) ? (long)M * (N / 2) : (long)M * N;
  int blocks = (int)std::min<long>((total + 255) / 256, 4096);
  hipLaunchKernelGGL((gemm_reduce_kernel<EPI, TR, TC>), dim3(blocks), dim3(256), 0, st, part, (const TR*)R, (TC*)C,
                     M, N, S);
  return 0;
}

// Skinny launch plan: WN 64-row blocks per workgroup and S K-splits. Two
// blocks per workgroup halve the activation traffic per weight byte and win
// whenever the grid still reaches ~160 workgroups; otherwise one block. The
// split count doubles until the grid reaches its target, while each split
// keeps at least 16 stages (shorter splits lose more to ring fill and
// drain than they gain in parallelism, and add partial-sum traffic).
// Chosen from a sweep of both widths and 1..8 splits over the 8B and 70B
// decode shapes at M = 32 and 64, reduction included.
static int skinny_splits_for(int tiles, int K, int target) {
  using namespace skinny;
  int S = 1;
  while (tiles * S < target && (K % (KS * S * 2)) == 0 && K / (S * 2) >= 16 * KS) S *= 2;
  return S;
}

SkinnyPlan gemm_skinny_plan(int M, int N, int K) {
  (void)M;
  if (N % 128 == 0) {
    const int S = skinny_splits_for(N / 128, K, 160);
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
                     st, (const bf16_t*)A, (const bf16_t*)W, part, (const TR*)R, (TC*)C, M, N, K, K / S);
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
  if ((pl.wn != 1 && pl.wn != 2) || N % (64 * pl.wn) != 0 || pl.s < 1 || K % (skinny::KS * pl.s) != 0) return -1;
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

}  // namespace ps

namespace ps {
// Host-side mirror of launch_gemm's dispatch conditions: 0 if supported.
int gemm_check(int dtype, int epi, int M, int N, int K) {
  if (M < 0 || N <= 0 || K <= 0) return -1;
  if (epi == 2 && N % (2 * kGateUpBlock) != 0) return -1;
  if (dtype == 0) return 0;
  if (dtype != 1 || K % 64 != 0) return -1;
  if (M <= skinny::MAXM && N % 64 == 0) return 0;
  return (N % 256 == 0) ? 0 : -1;
}
}  // namespace ps
