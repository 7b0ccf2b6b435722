// GEMMs of the layer: C = epilogue(A W^T), A [M, K], W [N, K] (both
// K-contiguous, the nn.Linear layout), fp32 accumulation (gfx950).
//
//  * gemm_tile_kernel: prefill-sized M. 256x256x64 workgroup tile, four waves
//    of 128x128, v_mfma_f32_32x32x16_bf16, operands staged through
//    double-buffered, XOR-swizzled LDS (128 KiB). MFMA-bound.
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

namespace ps {

__device__ __forceinline__ float silu_f(float x) { return x / (1.f + expf(-x)); }

template <typename T> __device__ __forceinline__ float ld_elt(const T* p, long i);
template <> __device__ __forceinline__ float ld_elt<float>(const float* p, long i) { return p[i]; }
template <> __device__ __forceinline__ float ld_elt<bf16_t>(const bf16_t* p, long i) { return bf2f(p[i]); }
template <typename T> __device__ __forceinline__ void st_elt(T* p, long i, float v);
template <> __device__ __forceinline__ void st_elt<float>(float* p, long i, float v) { p[i] = v; }
template <> __device__ __forceinline__ void st_elt<bf16_t>(bf16_t* p, long i, float v) { p[i] = f2bf(v); }

// ====================================================================== tile
namespace tile {
constexpr int BM = 256, BN = 256, BK = 64;
constexpr int NT = 256;                 // threads
constexpr int WTM = 128, WTN = 128;     // wave tile
constexpr int FM = WTM / 32, FN = WTN / 32;
constexpr int TILE_ELTS = BM * BK;      // per operand per stage
constexpr int LOADS = TILE_ELTS / 8 / NT;  // 16-byte loads per lane per operand per stage (8)

// element offset of (row, 16-byte chunk ch) in a swizzled [rows][64] tile
__device__ __forceinline__ int swz(int row, int ch) { return row * BK + ((ch ^ ((row >> 1) & 7)) << 3); }
}  // namespace tile

template <int EPI, typename TR, typename TC>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void gemm_tile_kernel(
    const bf16_t* __restrict__ A, const bf16_t* __restrict__ W, const TR* __restrict__ R, TC* __restrict__ C,
    int M, int N, int K, int tiles_n) {
  using namespace tile;
  extern __shared__ __attribute__((aligned(16))) bf16_t smem[];
  bf16_t* sA = smem;                      // [2][BM*BK]
  bf16_t* sB = smem + 2 * TILE_ELTS;      // [2][BN*BK]

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
  const int wm = wave >> 1, wn = wave & 1;
  const int g = lane >> 5, c = lane & 31;

  // Direct global->LDS loads (global_load_lds_dwordx4): one instruction of
  // a wave fills 1 KiB of LDS, lane l landing at +16*l, i.e. 8 rows of the
  // [rows][64] tile. Lane l therefore fetches the logical chunk that the
  // swizzle stores at its LDS position: row r = 8*i + l/8, position l%8,
  // chunk (l%8) ^ ((r >> 1) & 7). Wave w fills rows [64w, 64w + 64).
  const int lrow = lane >> 3, lpos = lane & 7;
  const bf16_t* ga[LOADS];
  const bf16_t* gb[LOADS];
#pragma unroll
  for (int i = 0; i < LOADS; ++i) {
    const int row = wave * 64 + i * 8 + lrow;
    const int ch = lpos ^ ((row >> 1) & 7);
    ga[i] = A + (long)min(m0 + row, M - 1) * K + ch * 8;
    gb[i] = W + (long)(n0 + row) * K + ch * 8;
  }
  auto gload = [&](int k0, int buf) {
    bf16_t* a = sA + buf * TILE_ELTS + wave * 64 * BK;
    bf16_t* b = sB + buf * TILE_ELTS + wave * 64 * BK;
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      __builtin_amdgcn_global_load_lds(ga[i] + k0, (__attribute__((address_space(3))) void*)(a + i * 8 * BK), 16, 0, 0);
      __builtin_amdgcn_global_load_lds(gb[i] + k0, (__attribute__((address_space(3))) void*)(b + i * 8 * BK), 16, 0, 0);
    }
  };

  f32x16_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int KT = K / BK;
  gload(0, 0);
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this wave's LDS fills landed
  __syncthreads();
  for (int kt = 0; kt < KT; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < KT) gload((kt + 1) * BK, buf ^ 1);
    const bf16_t* a = sA + buf * TILE_ELTS;
    const bf16_t* b = sB + buf * TILE_ELTS;
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      bf16x8_t af[FM], bfr[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i)
        af[i] = __builtin_bit_cast(bf16x8_t, *(const uint4*)(a + swz(wm * WTM + i * 32 + c, 2 * kk + g)));
#pragma unroll
      for (int j = 0; j < FN; ++j)
        bfr[j] = __builtin_bit_cast(bf16x8_t, *(const uint4*)(b + swz(wn * WTN + j * 32 + c, 2 * kk + g)));
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    __builtin_amdgcn_s_waitcnt(0x0F70);
    __syncthreads();
  }

  // epilogue: acc[i][j][r] = C[row 8(r/4) + 4g + r%4][col c] of block (i, j)
  const int rbase = m0 + wm * WTM, cbase = n0 + wn * WTN;
  if constexpr (EPI == 2) {
    const int ldc = N / 2;
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int jp = 0; jp < FN / 2; ++jp)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = rbase + i * 32 + 8 * (r >> 2) + 4 * g + (r & 3);
          if (row < M) {
            const int col = (cbase >> 1) + jp * 32 + c;
            st_elt<TC>(C, (long)row * ldc + col, silu_f(acc[i][2 * jp][r]) * acc[i][2 * jp + 1][r]);
          }
        }
  } else {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = rbase + i * 32 + 8 * (r >> 2) + 4 * g + (r & 3);
          if (row < M) {
            const long idx = (long)row * N + cbase + j * 32 + c;
            float v = acc[i][j][r];
            if constexpr (EPI == 1) v += ld_elt<TR>(R, idx);
            st_elt<TC>(C, idx, v);
          }
        }
  }
}

// ==================================================================== skinny
namespace skinny {
constexpr int NT = 256;
constexpr int BN = 64;        // columns per workgroup (16 per wave)
constexpr int KCH = 256;      // K chunk staged per step
constexpr int MAXM = 64;
// swizzled [64 rows][256] bf16 chunk: 32 16-byte chunks per row
__device__ __forceinline__ int swz(int row, int ch) { return row * KCH + ((ch ^ (row & 31)) << 3); }
}  // namespace skinny

template <int MB>
__global__ __launch_bounds__(256) void gemm_skinny_kernel(const bf16_t* __restrict__ A, const bf16_t* __restrict__ W,
                                                          float* __restrict__ part, int M, int N, int K,
                                                          int k_per_split) {
  using namespace skinny;
  __shared__ __attribute__((aligned(16))) bf16_t sA[2][MB * 16 * KCH];
  const int n0 = blockIdx.x * BN;
  const int split = blockIdx.y;
  const int kb = split * k_per_split;
  const int nch = k_per_split / KCH;
  const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
  const int g = lane >> 4, c = lane & 15;
  const int col = n0 + wave * 16 + c;
  const bf16_t* wrow = W + (long)col * K + 8 * g;

  constexpr int AL = MB * 16 * KCH / 8 / NT;  // 16-byte A loads per thread per chunk
  uint4 ra[AL];
  auto aload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < AL; ++i) {
      const int id = i * NT + t, row = id >> 5, ch = id & 31;
      ra[i] = (row < M) ? *(const uint4*)(A + (long)row * K + k0 + ch * 8) : make_uint4(0, 0, 0, 0);
    }
  };
  auto astore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < AL; ++i) {
      const int id = i * NT + t, row = id >> 5, ch = id & 31;
      *(uint4*)(&sA[buf][swz(row, ch)]) = ra[i];
    }
  };
  u32x4_t wc[KCH / 32], wn[KCH / 32];
  auto wload = [&](int k0, u32x4_t* w) {
#pragma unroll
    for (int j = 0; j < KCH / 32; ++j) w[j] = __builtin_nontemporal_load((const u32x4_t*)(wrow + k0 + 32 * j));
  };

  f32x4_t acc[MB];
#pragma unroll
  for (int i = 0; i < MB; ++i) acc[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  wload(kb, wc);
  aload(kb);
  astore(0);
  __syncthreads();
  for (int ci = 0; ci < nch; ++ci) {
    const int buf = ci & 1;
    const int knext = kb + (ci + 1) * KCH;
    if (ci + 1 < nch) {
      wload(knext, wn);
      aload(knext);
    }
#pragma unroll
    for (int j = 0; j < KCH / 32; ++j) {
      const bf16x8_t bw = __builtin_bit_cast(bf16x8_t, wc[j]);
#pragma unroll
      for (int i = 0; i < MB; ++i) {
        const bf16x8_t a = __builtin_bit_cast(bf16x8_t, *(const uint4*)(&sA[buf][swz(16 * i + c, 4 * j + g)]));
        acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, bw, acc[i], 0, 0, 0);
      }
    }
    if (ci + 1 < nch) {
      astore(buf ^ 1);
#pragma unroll
      for (int j = 0; j < KCH / 32; ++j) wc[j] = wn[j];
    }
    __syncthreads();
  }
  // acc[i][r] = partial C[16i + 4g + r][col]
  float* pp = part + (long)split * M * N;
#pragma unroll
  for (int i = 0; i < MB; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = 16 * i + 4 * g + r;
      if (row < M) pp[(long)row * N + col] = acc[i][r];
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
      sW[kk][r] = (n0 + r < N && k < K) ? W[(long)(n0 + r) * K + k] : 0.f;
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
static int launch_tile(int M, int N, int K, const void* A, const void* W, const void* R, void* C, hipStream_t st) {
  using namespace tile;
  const int tiles_m = (M + BM - 1) / BM, tiles_n = N / BN;
  const size_t lds = 4 * TILE_ELTS * sizeof(bf16_t);
  static const hipError_t attr = hipFuncSetAttribute((const void*)gemm_tile_kernel<EPI, TR, TC>,
                                                      hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (attr != hipSuccess) return -1;
  hipLaunchKernelGGL((gemm_tile_kernel<EPI, TR, TC>), dim3(tiles_m * tiles_n), dim3(NT), lds, st,
                     (const bf16_t*)A, (const bf16_t*)W, (const TR*)R, (TC*)C, M, N, K, tiles_n);
  return 0;
}

template <int EPI, typename TR, typename TC>
static int launch_reduce(int M, int N, int S, const float* part, const void* R, void* C, hipStream_t st) {
  const long total = (EPI == 2) ? (long)M * (N / 2) : (long)M * N;
  int blocks = (int)std::min<long>((total + 255) / 256, 4096);
  hipLaunchKernelGGL((gemm_reduce_kernel<EPI, TR, TC>), dim3(blocks), dim3(256), 0, st, part, (const TR*)R, (TC*)C,
                     M, N, S);
  return 0;
}

int gemm_skinny_splits(int M, int N, int K) {
  using namespace skinny;
  (void)M;
  const int tiles = N / BN;
  int S = 1;
  // enough workgroups to keep 256 CUs streaming, K chunks of KCH per split
  while (tiles * S < 512 && (K % (KCH * S * 2)) == 0 && K / (S * 2) >= 2 * KCH) S *= 2;
  return S;
}

static int launch_skinny_core(int M, int N, int K, int S, const void* A, const void* W, float* part, hipStream_t st) {
  using namespace skinny;
  dim3 grid(N / BN, S);
  const int kps = K / S;
  const int MB = (M + 15) / 16;
  switch (MB) {
    case 1: hipLaunchKernelGGL(gemm_skinny_kernel<1>, grid, dim3(NT), 0, st, (const bf16_t*)A, (const bf16_t*)W, part, M, N, K, kps); break;
    case 2: hipLaunchKernelGGL(gemm_skinny_kernel<2>, grid, dim3(NT), 0, st, (const bf16_t*)A, (const bf16_t*)W, part, M, N, K, kps); break;
    case 3: hipLaunchKernelGGL(gemm_skinny_kernel<3>, grid, dim3(NT), 0, st, (const bf16_t*)A, (const bf16_t*)W, part, M, N, K, kps); break;
    case 4: hipLaunchKernelGGL(gemm_skinny_kernel<4>, grid, dim3(NT), 0, st, (const bf16_t*)A, (const bf16_t*)W, part, M, N, K, kps); break;
    default: return -1;
  }
  return 0;
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
  return (size_t)gemm_skinny_splits(M, N, K) * M * N * sizeof(float);
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
  if (M <= skinny::MAXM && N % skinny::BN == 0 && K % skinny::KCH == 0) {
    const int S = gemm_skinny_splits(M, N, K);
    if (ws_bytes < (size_t)S * M * N * sizeof(float)) return -2;
    float* part = (float*)ws;
    if (launch_skinny_core(M, N, K, S, A, W, part, st)) return -1;
#define RED_CASE(E, TR_, TC_, rd, cd) \
  if (epi == E && r_dt == rd && c_dt == cd) return launch_reduce<E, TR_, TC_>(M, N, S, part, R, C, st);
    RED_CASE(0, float, bf16_t, 0, 1)
    RED_CASE(0, float, bf16_t, 1, 1)
    RED_CASE(0, float, float, 0, 0)
    RED_CASE(0, float, float, 1, 0)
    RED_CASE(1, bf16_t, float, 1, 0)
    RED_CASE(1, float, bf16_t, 0, 1)
    RED_CASE(1, bf16_t, bf16_t, 1, 1)
    RED_CASE(1, float, float, 0, 0)
    RED_CASE(2, float, bf16_t, 0, 1)
    RED_CASE(2, float, bf16_t, 1, 1)
    RED_CASE(2, float, float, 0, 0)
#undef RED_CASE
    return -1;
  }
  if (N % tile::BN != 0) return -1;
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
  if (M <= skinny::MAXM && N % skinny::BN == 0 && K % skinny::KCH == 0) return 0;
  return (N % tile::BN == 0) ? 0 : -1;
}
}  // namespace ps
