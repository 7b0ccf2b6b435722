// RMSNorm, RoPE + paged KV write, KV append and KV gather (gfx950).
//
// All four are HBM-bound streaming kernels: one row (token) per workgroup,
// fp32 arithmetic, coalesced row reads.
#include "common.h"
#include "launch.h"

#include <type_traits>

namespace ps {

// ---------------------------------------------------------------- RMSNorm
// y = x / sqrt(mean(x^2) + eps) * g, one row per 256-thread workgroup.
template <typename TX, typename TG, typename TY>
__global__ __launch_bounds__(256) void rmsnorm_kernel(const TX* __restrict__ x, const TG* __restrict__ g,
                                                      TY* __restrict__ y, int d, float eps) {
  const long row = blockIdx.x;
  const TX* xr = x + row * d;
  float ss = 0.f;
  for (int i = threadIdx.x; i < d; i += 256) {
    float v = Elt<TX>::load(xr, i);
    ss += v * v;
  }
  for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o);
  __shared__ float red[4];
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  float tot = red[0] + red[1] + red[2] + red[3];
  float inv = 1.0f / sqrtf(tot / (float)d + eps);
  TY* yr = y + row * d;
  for (int i = threadIdx.x; i < d; i += 256) {
    Elt<TY>::store(yr, i, Elt<TX>::load(xr, i) * inv * Elt<TG>::load(g, i));
  }
}

// Second half of the vectorised RMSNorm, shared by the kernels that hold a
// row in registers (v[c][e] = element (c * 256 + threadIdx.x) * 8 + e):
// sum of squares in that order, wave then workgroup reduction, bf16 output.
template <int VPT>
__device__ __forceinline__ void rmsnorm_row_out(const float (&v)[VPT][8], const bf16_t* __restrict__ g,
                                                bf16_t* __restrict__ yr, int d, float eps) {
  float ss = 0.f;
#pragma unroll
  for (int c = 0; c < VPT; ++c) {
    const int i = (c * 256 + threadIdx.x) * 8;
    if (i < d) {
#pragma unroll
      for (int e = 0; e < 8; ++e) ss += v[c][e] * v[c][e];
    }
  }
  for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o);
  __shared__ float red[4];
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  float tot = red[0] + red[1] + red[2] + red[3];
  float inv = 1.0f / sqrtf(tot / (float)d + eps);
#pragma unroll
  for (int c = 0; c < VPT; ++c) {
    int i = (c * 256 + threadIdx.x) * 8;
    if (i < d) {
      uint4 gw = *(const uint4*)(g + i);
      uint32_t gs[4] = {gw.x, gw.y, gw.z, gw.w};
      uint32_t o[4];
#pragma unroll
      for (int e = 0; e < 4; ++e)
        o[e] = pack_bf2(v[c][2 * e] * inv * bf_lo(gs[e]), v[c][2 * e + 1] * inv * bf_hi(gs[e]));
      *(uint4*)(yr + i) = make_uint4(o[0], o[1], o[2], o[3]);
    }
  }
}

// Vectorised bf16 -> bf16 variant: 8 elements per 16-byte access, the row
// kept in registers between the two passes (d <= 256 * 8 * VPT).
// The first up.blocks workgroups carry a metadata upload instead (the first
// kernel of a layer call takes its call's upload along, saving a launch).
template <typename TX, int VPT>
__global__ __launch_bounds__(256) void rmsnorm_vec_kernel(const TX* __restrict__ x, const bf16_t* __restrict__ g,
                                                          bf16_t* __restrict__ y, int d, float eps, UploadJob up) {
  if ((int)blockIdx.x < up.blocks) {
    upload_block(up, blockIdx.x);
    return;
  }
  const long row = blockIdx.x - up.blocks;
  float v[VPT][8];
#pragma unroll
  for (int c = 0; c < VPT; ++c) {
    int i = (c * 256 + threadIdx.x) * 8;
    if (i < d) {
      if constexpr (sizeof(TX) == 2) {
        uint4 w = *(const uint4*)(x + row * d + i);
        uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          v[c][2 * e] = bf_lo(ws[e]);
          v[c][2 * e + 1] = bf_hi(ws[e]);
        }
      } else {
        float4 a = *(const float4*)(x + row * d + i);
        float4 b = *(const float4*)(x + row * d + i + 4);
        v[c][0] = a.x; v[c][1] = a.y; v[c][2] = a.z; v[c][3] = a.w;
        v[c][4] = b.x; v[c][5] = b.y; v[c][6] = b.z; v[c][7] = b.w;
      }
    }
  }
  rmsnorm_row_out<VPT>(v, g, y + row * d, d, eps);
}

// Decode-sized O projection fused with its consumer: h = sum of the split-K
// partials of o W^T, in split order, + the residual x (bf16), stored fp32;
// then hn = RMSNorm(h) * g from the same registers. The sum and the norm
// are those of the separate reduce and RMSNorm kernels, bit for bit.
template <int VPT, int S>
__global__ __launch_bounds__(256) void split_residual_rmsnorm_kernel(const float* __restrict__ part, long mn,
                                                                     const bf16_t* __restrict__ res,
                                                                     float* __restrict__ h,
                                                                     const bf16_t* __restrict__ g,
                                                                     bf16_t* __restrict__ y, int d, float eps) {
  const long row = blockIdx.x;
  float v[VPT][8];
  // every partial and residual load of the row is issued before the sums
  // (S is a compile-time count): one round of memory latency, not S x VPT
  float4 pa[VPT][S][2];
  uint4 rw[VPT];
#pragma unroll
  for (int c = 0; c < VPT; ++c) {
    const int i = (c * 256 + threadIdx.x) * 8;
    if (i < d) {
      const long off = row * d + i;
#pragma unroll
      for (int sp = 0; sp < S; ++sp) {
        pa[c][sp][0] = *(const float4*)(part + sp * mn + off);
        pa[c][sp][1] = *(const float4*)(part + sp * mn + off + 4);
      }
      rw[c] = *(const uint4*)(res + off);
    }
  }
#pragma unroll
  for (int c = 0; c < VPT; ++c) {
    const int i = (c * 256 + threadIdx.x) * 8;
    if (i < d) {
#pragma unroll
      for (int e = 0; e < 8; ++e) v[c][e] = 0.f;
#pragma unroll
      for (int sp = 0; sp < S; ++sp) {
        v[c][0] += pa[c][sp][0].x; v[c][1] += pa[c][sp][0].y; v[c][2] += pa[c][sp][0].z; v[c][3] += pa[c][sp][0].w;
        v[c][4] += pa[c][sp][1].x; v[c][5] += pa[c][sp][1].y; v[c][6] += pa[c][sp][1].z; v[c][7] += pa[c][sp][1].w;
      }
      const uint32_t rs[4] = {rw[c].x, rw[c].y, rw[c].z, rw[c].w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[c][2 * e] += bf_lo(rs[e]);
        v[c][2 * e + 1] += bf_hi(rs[e]);
      }
      const long off = row * d + i;
      *(float4*)(h + off) = make_float4(v[c][0], v[c][1], v[c][2], v[c][3]);
      *(float4*)(h + off + 4) = make_float4(v[c][4], v[c][5], v[c][6], v[c][7]);
    }
  }
  rmsnorm_row_out<VPT>(v, g, y + row * d, d, eps);
}

int launch_split_residual_rmsnorm(int rows, int d, int S, const float* part, const void* res, float* h,
                                  const void* g, float eps, void* y, hipStream_t st) {
  if (rows == 0) return 0;
  if (d % 8 != 0 || d > 256 * 8 * 4) return -1;
  const long mn = (long)rows * d;
#define SRR_CASE(S_)                                                                                        \
  if (S == S_) {                                                                                            \
    hipLaunchKernelGGL((split_residual_rmsnorm_kernel<4, S_>), dim3(rows), dim3(256), 0, st, part, mn,       \
                       (const bf16_t*)res, h, (const bf16_t*)g, (bf16_t*)y, d, eps);                        \
    return 0;                                                                                               \
  }
  SRR_CASE(2)
  SRR_CASE(3)
  SRR_CASE(4)
  SRR_CASE(8)
#undef SRR_CASE
  return -1;
}

bool rmsnorm_carries_upload(int x_dt, int g_dt, int y_dt, int d) {
  (void)x_dt;
  return g_dt == 1 && y_dt == 1 && d % 8 == 0 && d <= 256 * 8 * 4;
}

int launch_rmsnorm(int x_dt, int g_dt, int y_dt, int rows, int d, const void* x, const void* g, float eps,
                   void* y, hipStream_t st, const UploadJob* up) {
  if (rmsnorm_carries_upload(x_dt, g_dt, y_dt, d)) {
    const UploadJob j = up ? *up : UploadJob{};
    if (rows + j.blocks == 0) return 0;
    dim3 grid(rows + j.blocks), block(256);
    if (x_dt == 1) {
      hipLaunchKernelGGL((rmsnorm_vec_kernel<bf16_t, 4>), grid, block, 0, st, (const bf16_t*)x,
                         (const bf16_t*)g, (bf16_t*)y, d, eps, j);
    } else {
      hipLaunchKernelGGL((rmsnorm_vec_kernel<float, 4>), grid, block, 0, st, (const float*)x,
                         (const bf16_t*)g, (bf16_t*)y, d, eps, j);
    }
    return 0;
  }
  if (up && launch_upload(*up, st)) return -1;
  if (rows == 0) return 0;
  dim3 grid(rows), block(256);
#define RMS_CASE(TX_, TG_, TY_, a, b, c)                                                           \
  if (x_dt == a && g_dt == b && y_dt == c) {                                                       \
    hipLaunchKernelGGL((rmsnorm_kernel<TX_, TG_, TY_>), grid, block, 0, st, (const TX_*)x,        \
                       (const TG_*)g, (TY_*)y, d, eps);                                           \
    return 0;                                                                                      \
  }
  RMS_CASE(float, float, float, 0, 0, 0)
  RMS_CASE(float, float, bf16_t, 0, 0, 1)
  RMS_CASE(bf16_t, bf16_t, bf16_t, 1, 1, 1)
  RMS_CASE(bf16_t, bf16_t, float, 1, 1, 0)
  RMS_CASE(float, bf16_t, bf16_t, 0, 1, 1)
  RMS_CASE(float, bf16_t, float, 0, 1, 0)
  RMS_CASE(bf16_t, float, float, 1, 0, 0)
  RMS_CASE(bf16_t, float, bf16_t, 1, 0, 1)
#undef RMS_CASE
  return -1;
}

// ---------------------------------------------------------------- paging
// Element offset of the K row of (page, kv head, slot) within a layer, and
// of the V^T column. Page block per (page, kv head): K [16][hd] then
// V^T [hd][16].
__device__ __forceinline__ long kv_block(int page, int kvh, int n_kv, int hd) {
  return ((long)page * n_kv + kvh) * (2L * kPageTokens * hd);
}

__device__ __forceinline__ int find_seq(const SeqInfo* __restrict__ si, int n_seqs, int row) {
  int lo = 0, hi = n_seqs - 1;
  while (lo < hi) {  // last b with row_start <= row
    int mid = (lo + hi + 1) >> 1;
    if (si[mid].row_start <= row) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// The same search by one whole wave: each round loads 64 row_starts in
// parallel and counts those <= row, so n sequences take ceil(log64 n) load
// round trips instead of log2 n dependent ones. Every lane gets the result.
__device__ __forceinline__ int find_seq_wave(const SeqInfo* __restrict__ si, int n_seqs, int row) {
  const int lane = threadIdx.x & 63;
  int lo = 0, n = n_seqs;
  while (n > 64) {
    const int stride = (n + 63) / 64;
    const int idx = lo + lane * stride;
    const bool le = idx < lo + n && si[idx].row_start <= row;
    const int cnt = __popcll(__ballot(le));  // >= 1: si[lo].row_start <= row
    lo += (cnt - 1) * stride;
    n = min(stride, n - (cnt - 1) * stride);
  }
  const bool le = lane < n && si[lo + lane].row_start <= row;
  return lo + __popcll(__ballot(le)) - 1;
}

// ---------------------------------------------------------------- RoPE + KV
// One row per workgroup: rotate the row's q and k heads (rotate-half, angle
// pos * inv_freq[j] evaluated in fp64), write q to q_out and k, v into the
// row's page slot. bf16 rows move four pairs per thread with 8-byte accesses.
// PART (bf16, decode): the QKV row is not materialised; it is the sum of the
// GEMM's S split-K partials (fp32 [S][rows][n_q + 2 n_kv][hd]) in split order,
// rounded to bf16, exactly what the separate reduce kernel would have stored.
template <typename T, int SS>
__global__ __launch_bounds__(256) void rope_kvwrite_kernel(const T* __restrict__ qkv, T* __restrict__ q_out,
                                                           T* __restrict__ pool, const SeqInfo* __restrict__ si,
                                                           const int32_t* __restrict__ bt,
                                                           const double* __restrict__ inv_freq, int n_seqs,
                                                           int n_q, int n_kv, int hd, const float* __restrict__ part,
                                                           long mn) {
  constexpr bool PART = SS > 0;  // SS split-K partials, a compile-time count
  static_assert(!PART || std::is_same<T, bf16_t>::value, "split partials feed the bf16 path");
  const int row = blockIdx.x;
  const int half = hd >> 1;
  __shared__ float cs[64], sn[64];
  __shared__ int s_b;
  if (threadIdx.x < 64) {
    const int b = find_seq_wave(si, n_seqs, row);
    if (threadIdx.x == 0) s_b = b;
  }
  __syncthreads();
  const SeqInfo s = si[s_b];
  const int pos = s.kv_before + (row - s.row_start);
  for (int j = threadIdx.x; j < half; j += blockDim.x) {
    double a = (double)pos * inv_freq[j];
    double sv, cv;
    sincos(a, &sv, &cv);
    cs[j] = (float)cv;
    sn[j] = (float)sv;
  }
  __syncthreads();
  const int dqkv = (n_q + 2 * n_kv) * hd;
  const T* xr = qkv + (long)row * dqkv;
  const float* pr = PART ? part + (long)row * dqkv : nullptr;  // partials of this row
  // four consecutive elements of the row from column col (col % 4 == 0)
  auto load4 = [&](int col, float (&x)[4]) {
    if constexpr (PART) {
      float4 p4[SS > 0 ? SS : 1];
#pragma unroll
      for (int sp = 0; sp < SS; ++sp) p4[sp] = *(const float4*)(pr + sp * mn + col);
      float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
      for (int sp = 0; sp < SS; ++sp) {
        acc.x += p4[sp].x; acc.y += p4[sp].y; acc.z += p4[sp].z; acc.w += p4[sp].w;
      }
      x[0] = bf2f(f2bf(acc.x)); x[1] = bf2f(f2bf(acc.y)); x[2] = bf2f(f2bf(acc.z)); x[3] = bf2f(f2bf(acc.w));
    } else {
      const uint2 a = *(const uint2*)(xr + col);
      x[0] = bf_lo(a.x); x[1] = bf_hi(a.x); x[2] = bf_lo(a.y); x[3] = bf_hi(a.y);
    }
  };
  auto load1 = [&](int col) -> float {
    if constexpr (PART) {
      float p1[SS > 0 ? SS : 1];
#pragma unroll
      for (int sp = 0; sp < SS; ++sp) p1[sp] = pr[sp * mn + col];
      float acc = 0.f;
#pragma unroll
      for (int sp = 0; sp < SS; ++sp) acc += p1[sp];
      return bf2f(f2bf(acc));
    } else {
      return Elt<T>::load(xr, col);
    }
  };
  const int page = bt[s.bt_off + pos / kPageTokens];
  const int slot = pos % kPageTokens;
  auto dst_of = [&](int head) -> T* {  // start of the head's rotated row
    return head < n_q ? q_out + (long)row * n_q * hd + head * hd
                      : pool + kv_block(page, head - n_q, n_kv, hd) + (long)slot * hd;
  };
  bool quad = false;
  if constexpr (std::is_same<T, bf16_t>::value) quad = (half % 4) == 0;
  if (quad) {
    // q and k: pairs (j, j + half), four consecutive j per thread (hd % 8 == 0)
    const int quads = half / 4;
    for (int idx = threadIdx.x; idx < (n_q + n_kv) * quads; idx += blockDim.x) {
      const int head = idx / quads, j = (idx - head * quads) * 4;
      float x1[4], x2[4];
      load4(head * hd + j, x1);
      load4(head * hd + j + half, x2);
      float y1[4], y2[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        y1[e] = x1[e] * cs[j + e] - x2[e] * sn[j + e];
        y2[e] = x2[e] * cs[j + e] + x1[e] * sn[j + e];
      }
      T* d = dst_of(head);
      *(uint2*)(d + j) = make_uint2(pack_bf2(y1[0], y1[1]), pack_bf2(y1[2], y1[3]));
      *(uint2*)(d + j + half) = make_uint2(pack_bf2(y2[0], y2[1]), pack_bf2(y2[2], y2[3]));
    }
  } else {
    for (int idx = threadIdx.x; idx < (n_q + n_kv) * half; idx += blockDim.x) {
      int head = idx / half, j = idx - head * half;
      float x1 = load1(head * hd + j);
      float x2 = load1(head * hd + j + half);
      T* d = dst_of(head);
      Elt<T>::store(d, j, x1 * cs[j] - x2 * sn[j]);
      Elt<T>::store(d, j + half, x2 * cs[j] + x1 * sn[j]);
    }
  }
  // v: stored dimension-major within the page
  if constexpr (PART) {
    // four consecutive dimensions per thread (hd % 4 == 0 on the bf16 path)
    for (int idx = threadIdx.x * 4; idx < n_kv * hd; idx += blockDim.x * 4) {
      const int kvh = idx / hd, dim = idx - kvh * hd;
      float x4[4];
      load4((n_q + n_kv) * hd + idx, x4);
      T* vb = pool + kv_block(page, kvh, n_kv, hd) + (long)kPageTokens * hd + slot;
#pragma unroll
      for (int e = 0; e < 4; ++e) vb[(long)(dim + e) * kPageTokens] = f2bf(x4[e]);
    }
  } else {
    for (int idx = threadIdx.x; idx < n_kv * hd; idx += blockDim.x) {
      int kvh = idx / hd, dim = idx - kvh * hd;
      T v = xr[(n_q + n_kv) * hd + idx];
      pool[kv_block(page, kvh, n_kv, hd) + (long)kPageTokens * hd + (long)dim * kPageTokens + slot] = v;
    }
  }
}

// Prefill-sized bf16 RoPE + KV write: 16 rows per workgroup of 1024 threads
// (a page's worth of tokens; about one sequence lookup per wave and one angle
// per thread), the same arithmetic per element as rope_kvwrite_kernel. q and k
// move eight pairs per thread with 16-byte accesses. v is staged through LDS:
// when the 16 rows are one sequence's positions p0 .. p0+15 with p0 % 16 == 0
// (they fill one page), each thread writes one dimension's 16 slots of the
// dimension-major page as two 16-byte stores; otherwise 2-byte stores.
constexpr int kRopeRows = 16;
__global__ __launch_bounds__(1024) void rope_kvwrite_rows_kernel(const bf16_t* __restrict__ qkv,
                                                                bf16_t* __restrict__ q_out, bf16_t* __restrict__ pool,
                                                                const SeqInfo* __restrict__ si,
                                                                const int32_t* __restrict__ bt,
                                                                const double* __restrict__ inv_freq, int rows,
                                                                int n_seqs, int n_q, int n_kv, int hd) {
  constexpr int RB = kRopeRows;
  const int row0 = blockIdx.x * RB;
  const int nr = min(RB, rows - row0);
  const int half = hd >> 1;  // <= 64, a multiple of 8
  const int dqkv = (n_q + 2 * n_kv) * hd;
  const int vcols = n_kv * hd;
  __shared__ float cs[RB][64], sn[RB][64];
  __shared__ int s_b[RB], s_pos[RB], s_page[RB];
  extern __shared__ __attribute__((aligned(16))) bf16_t sv[];  // [RB][vcols]
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, n_waves = blockDim.x >> 6;
  for (int r = wave; r < nr; r += n_waves) {
    const int b = find_seq_wave(si, n_seqs, row0 + r);
    if (lane == 0) {
      const SeqInfo sq = si[b];
      const int pos = sq.kv_before + (row0 + r - sq.row_start);
      s_b[r] = b;
      s_pos[r] = pos;
      s_page[r] = bt[sq.bt_off + pos / kPageTokens];
    }
  }
  // v rows of the block into LDS, 16 bytes per thread
  const int vchunks = vcols / 8;
  for (int idx = threadIdx.x; idx < nr * vchunks; idx += blockDim.x) {
    const int r = idx / vchunks, ch = idx - r * vchunks;
    *(uint4*)(sv + r * vcols + ch * 8) = *(const uint4*)(qkv + (long)(row0 + r) * dqkv + (n_q + n_kv) * hd + ch * 8);
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < nr * half; idx += blockDim.x) {
    const int r = idx / half, j = idx - r * half;
    double a = (double)s_pos[r] * inv_freq[j];
    double sv_, cv;
    sincos(a, &sv_, &cv);
    cs[r][j] = (float)cv;
    sn[r][j] = (float)sv_;
  }
  __syncthreads();
  // q and k: pairs (j, j + half), eight consecutive j per thread
  const int octs = half / 8;
  const int per_row = (n_q + n_kv) * octs;
  for (int idx = threadIdx.x; idx < nr * per_row; idx += blockDim.x) {
    const int r = idx / per_row, rem = idx - r * per_row;
    const int head = rem / octs, j = (rem - head * octs) * 8;
    const bf16_t* xr = qkv + (long)(row0 + r) * dqkv + head * hd;
    const uint4 a1 = *(const uint4*)(xr + j), a2 = *(const uint4*)(xr + j + half);
    const uint32_t w1[4] = {a1.x, a1.y, a1.z, a1.w}, w2[4] = {a2.x, a2.y, a2.z, a2.w};
    uint32_t o1[4], o2[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float x1l = bf_lo(w1[e]), x1h = bf_hi(w1[e]), x2l = bf_lo(w2[e]), x2h = bf_hi(w2[e]);
      const float cl = cs[r][j + 2 * e], ch = cs[r][j + 2 * e + 1], sl = sn[r][j + 2 * e], sh = sn[r][j + 2 * e + 1];
      o1[e] = pack_bf2(x1l * cl - x2l * sl, x1h * ch - x2h * sh);
      o2[e] = pack_bf2(x2l * cl + x1l * sl, x2h * ch + x1h * sh);
    }
    bf16_t* d = head < n_q ? q_out + ((long)(row0 + r) * n_q + head) * hd
                           : pool + kv_block(s_page[r], head - n_q, n_kv, hd) + (long)(s_pos[r] % kPageTokens) * hd;
    *(uint4*)(d + j) = make_uint4(o1[0], o1[1], o1[2], o1[3]);
    *(uint4*)(d + j + half) = make_uint4(o2[0], o2[1], o2[2], o2[3]);
  }
  // v: dimension-major within the page
  const bool one_page = nr == RB && s_b[0] == s_b[RB - 1] && s_pos[0] % kPageTokens == 0;
  if (one_page) {
    for (int idx = threadIdx.x; idx < vcols; idx += blockDim.x) {
      const int kvh = idx / hd, dim = idx - kvh * hd;
      uint32_t w[8];
#pragma unroll
      for (int e = 0; e < 8; ++e)
        w[e] = (uint32_t)__builtin_bit_cast(uint16_t, sv[(2 * e) * vcols + idx]) |
               ((uint32_t)__builtin_bit_cast(uint16_t, sv[(2 * e + 1) * vcols + idx]) << 16);
      bf16_t* vb = pool + kv_block(s_page[0], kvh, n_kv, hd) + (long)kPageTokens * hd + (long)dim * kPageTokens;
      *(uint4*)vb = make_uint4(w[0], w[1], w[2], w[3]);
      *(uint4*)(vb + 8) = make_uint4(w[4], w[5], w[6], w[7]);
    }
  } else {
    for (int idx = threadIdx.x; idx < nr * vcols; idx += blockDim.x) {
      const int r = idx / vcols, c = idx - r * vcols;
      const int kvh = c / hd, dim = c - kvh * hd;
      pool[kv_block(s_page[r], kvh, n_kv, hd) + (long)kPageTokens * hd + (long)dim * kPageTokens +
           s_pos[r] % kPageTokens] = sv[r * vcols + c];
    }
  }
}

int launch_rope_kvwrite(int dt, int rows, const void* qkv, void* q_out, void* pool_layer, const SeqInfo* si,
                        const int32_t* bt, const double* inv_freq, int n_seqs, int n_q, int n_kv, int hd,
                        hipStream_t st, const float* part, int splits) {
  if (rows == 0) return 0;
  if (hd > 128) return -1;
  const long mn = (long)rows * (n_q + 2 * n_kv) * hd;
  if (part && splits > 1) {
    if (dt != 1 || hd % 8 != 0) return -1;
#define ROPE_PART_CASE(S_)                                                                                      \
    if (splits == S_) {                                                                                         \
      hipLaunchKernelGGL((rope_kvwrite_kernel<bf16_t, S_>), dim3(rows), dim3(256), 0, st, (const bf16_t*)qkv,   \
                         (bf16_t*)q_out, (bf16_t*)pool_layer, si, bt, inv_freq, n_seqs, n_q, n_kv, hd, part, mn); \
      return 0;                                                                                                 \
    }
    ROPE_PART_CASE(2)
    ROPE_PART_CASE(3)
    ROPE_PART_CASE(4)
    ROPE_PART_CASE(8)
#undef ROPE_PART_CASE
    return -1;
  }
  const size_t v_lds = (size_t)kRopeRows * n_kv * hd * sizeof(bf16_t);
  if (dt == 1 && hd % 16 == 0 && v_lds <= 64 * 1024) {
    static const hipError_t attr = hipFuncSetAttribute((const void*)rope_kvwrite_rows_kernel,
                                                       hipFuncAttributeMaxDynamicSharedMemorySize, 64 * 1024);
    if (attr != hipSuccess) return -1;
    hipLaunchKernelGGL(rope_kvwrite_rows_kernel, dim3((rows + kRopeRows - 1) / kRopeRows), dim3(1024), v_lds, st,
                       (const bf16_t*)qkv, (bf16_t*)q_out, (bf16_t*)pool_layer, si, bt, inv_freq, rows, n_seqs, n_q,
                       n_kv, hd);
  } else if (dt == 1)
    hipLaunchKernelGGL((rope_kvwrite_kernel<bf16_t, 0>), dim3(rows), dim3(256), 0, st, (const bf16_t*)qkv,
                       (bf16_t*)q_out, (bf16_t*)pool_layer, si, bt, inv_freq, n_seqs, n_q, n_kv, hd, nullptr, 0L);
  else
    hipLaunchKernelGGL((rope_kvwrite_kernel<float, 0>), dim3(rows), dim3(256), 0, st, (const float*)qkv,
                       (float*)q_out, (float*)pool_layer, si, bt, inv_freq, n_seqs, n_q, n_kv, hd, nullptr, 0L);
  return 0;
}

// ---------------------------------------------------------------- append
// Caller K/V rows [rows, n_kv, hd] into their page slots (no rotation).
template <typename T>
__global__ __launch_bounds__(256) void kv_append_kernel(const T* __restrict__ k, const T* __restrict__ v,
                                                        T* __restrict__ pool, const SeqInfo* __restrict__ si,
                                                        const int32_t* __restrict__ bt, int n_seqs, int n_kv,
                                                        int hd) {
  const int row = blockIdx.x;
  __shared__ int s_b;
  if (threadIdx.x < 64) {
    const int b = find_seq_wave(si, n_seqs, row);
    if (threadIdx.x == 0) s_b = b;
  }
  __syncthreads();
  const SeqInfo s = si[s_b];
  const int pos = s.kv_before + (row - s.row_start);
  const int page = bt[s.bt_off + pos / kPageTokens];
  const int slot = pos % kPageTokens;
  for (int idx = threadIdx.x; idx < n_kv * hd; idx += blockDim.x) {
    int kvh = idx / hd, dim = idx - kvh * hd;
    long base = kv_block(page, kvh, n_kv, hd);
    pool[base + (long)slot * hd + dim] = k[(long)row * n_kv * hd + idx];
    pool[base + (long)kPageTokens * hd + (long)dim * kPageTokens + slot] = v[(long)row * n_kv * hd + idx];
  }
}

int launch_kv_append(int dt, int rows, const void* k, const void* v, void* pool_layer, const SeqInfo* si,
                     const int32_t* bt, int n_seqs, int n_kv, int hd, hipStream_t st) {
  if (rows == 0) return 0;
  if (dt == 1)
    hipLaunchKernelGGL(kv_append_kernel<bf16_t>, dim3(rows), dim3(256), 0, st, (const bf16_t*)k,
                       (const bf16_t*)v, (bf16_t*)pool_layer, si, bt, n_seqs, n_kv, hd);
  else
    hipLaunchKernelGGL(kv_append_kernel<float>, dim3(rows), dim3(256), 0, st, (const float*)k,
                       (const float*)v, (float*)pool_layer, si, bt, n_seqs, n_kv, hd);
  return 0;
}

// ---------------------------------------------------------------- gather
// Positions [0, len) of one sequence into contiguous [len, n_kv, hd].
template <typename T>
__global__ __launch_bounds__(256) void kv_gather_kernel(const T* __restrict__ pool, const int32_t* __restrict__ bt,
                                                        T* __restrict__ k_out, T* __restrict__ v_out, int n_kv,
                                                        int hd) {
  const int pos = blockIdx.x;
  const int page = bt[pos / kPageTokens];
  const int slot = pos % kPageTokens;
  for (int idx = threadIdx.x; idx < n_kv * hd; idx += blockDim.x) {
    int kvh = idx / hd, dim = idx - kvh * hd;
    long base = kv_block(page, kvh, n_kv, hd);
    k_out[(long)pos * n_kv * hd + idx] = pool[base + (long)slot * hd + dim];
    v_out[(long)pos * n_kv * hd + idx] = pool[base + (long)kPageTokens * hd + (long)dim * kPageTokens + slot];
  }
}

int launch_kv_gather(int dt, int len, const void* pool_layer, const int32_t* bt, void* k_out, void* v_out,
                     int n_kv, int hd, hipStream_t st) {
  if (len == 0) return 0;
  if (dt == 1)
    hipLaunchKernelGGL(kv_gather_kernel<bf16_t>, dim3(len), dim3(256), 0, st, (const bf16_t*)pool_layer, bt,
                       (bf16_t*)k_out, (bf16_t*)v_out, n_kv, hd);
  else
    hipLaunchKernelGGL(kv_gather_kernel<float>, dim3(len), dim3(256), 0, st, (const float*)pool_layer, bt,
                       (float*)k_out, (float*)v_out, n_kv, hd);
  return 0;
}

// ---------------------------------------------------------------- transfer
// Whole pages of one sequence, every layer, from one pool to another: block
// (p, l) copies logical page p of layer l (all KV heads, K and V^T) from the
// source's physical page src_bt[p] to the destination's dst_bt[p]. Pools may
// have different page counts, hence their own layer strides. 16-byte copies.
__global__ __launch_bounds__(256) void kv_copy_pages_kernel(const uint4* __restrict__ src, long src_layer16,
                                                            const int32_t* __restrict__ src_bt,
                                                            uint4* __restrict__ dst, long dst_layer16,
                                                            const int32_t* __restrict__ dst_bt, int page16) {
  const int p = blockIdx.x, l = blockIdx.y;
  const uint4* s = src + l * src_layer16 + (long)src_bt[p] * page16;
  uint4* d = dst + l * dst_layer16 + (long)dst_bt[p] * page16;
  for (int i = threadIdx.x; i < page16; i += 256) d[i] = s[i];
}

int launch_kv_copy_pages(size_t page_bytes, int n_pages, int n_layers, const void* src_pool, size_t src_layer_bytes,
                         const int32_t* src_bt, void* dst_pool, size_t dst_layer_bytes, const int32_t* dst_bt,
                         hipStream_t st) {
  if (n_pages == 0 || n_layers == 0) return 0;
  if (page_bytes % 16 || src_layer_bytes % 16 || dst_layer_bytes % 16 || n_layers > 65535) return -1;
  hipLaunchKernelGGL(kv_copy_pages_kernel, dim3(n_pages, n_layers), dim3(256), 0, st, (const uint4*)src_pool,
                     (long)(src_layer_bytes / 16), src_bt, (uint4*)dst_pool, (long)(dst_layer_bytes / 16), dst_bt,
                     (int)(page_bytes / 16));
  return 0;
}

}  // namespace ps
