// Model-level kernels (gfx950): embedding gather, row gather, greedy argmax.
#include "common.h"
#include "launch.h"

#include <algorithm>

namespace ps {

// x[r, :] = table[tokens[r], :], 16 bytes per thread.
// Token ids outside [0, vocab) embed as zero rows (ids live on the device,
// so they cannot be validated on the host before the launch).
__global__ __launch_bounds__(256) void embed_kernel(const bf16_t* __restrict__ table, const int32_t* __restrict__ tokens,
                                                    bf16_t* __restrict__ x, int d, int vocab) {
  const long r = blockIdx.x;
  const int tok = tokens[r];
  if (tok < 0 || tok >= vocab) {
    for (int i = threadIdx.x * 8; i < d; i += 256 * 8) *(uint4*)(x + r * d + i) = make_uint4(0, 0, 0, 0);
    return;
  }
  for (int i = threadIdx.x * 8; i < d; i += 256 * 8)
    *(uint4*)(x + r * d + i) = *(const uint4*)(table + (long)tok * d + i);
}

// dst[i, :] = src[rows[i], :] (bf16 rows of d elements)
__global__ __launch_bounds__(256) void gather_rows_kernel(const bf16_t* __restrict__ src, const int32_t* __restrict__ rows,
                                                          bf16_t* __restrict__ dst, int d) {
  const long i = blockIdx.x;
  const long r = rows[i];
  for (int e = threadIdx.x * 8; e < d; e += 256 * 8) *(uint4*)(dst + i * d + e) = *(const uint4*)(src + r * d + e);
}

// next[r] = argmax_j logits[r, j], ties to the lowest j. One workgroup of
// 1024 threads per row, 16-byte loads where the row allows (a decode step has
// only as many rows as sequences, so each row needs many loads in flight).
// NaN never compares greater; an all-NaN row gives 0.
constexpr int kArgmaxThreads = 1024;
__global__ __launch_bounds__(kArgmaxThreads) void argmax_kernel(const float* __restrict__ logits,
                                                                int32_t* __restrict__ next, int vocab) {
  const long r = blockIdx.x;
  const float* row = logits + r * vocab;
  float best = -INFINITY;
  int bi = 0x7fffffff;
  // each thread visits its indices in increasing order, and "strictly
  // greater" then keeps the lowest index among equal values
  if (vocab % 4 == 0 && ((uintptr_t)row & 15) == 0) {
    const int n4 = vocab / 4;
#pragma unroll 4
    for (int j4 = threadIdx.x; j4 < n4; j4 += kArgmaxThreads) {
      const float4 v = *(const float4*)(row + 4 * (long)j4);
      const int j = 4 * j4;
      if (v.x > best) { best = v.x; bi = j; }
      if (v.y > best) { best = v.y; bi = j + 1; }
      if (v.z > best) { best = v.z; bi = j + 2; }
      if (v.w > best) { best = v.w; bi = j + 3; }
    }
  } else {
    for (int j = threadIdx.x; j < vocab; j += kArgmaxThreads) {
      const float v = row[j];
      if (v > best) {
        best = v;
        bi = j;
      }
    }
  }
  for (int off = 32; off > 0; off >>= 1) {
    const float ov = __shfl_xor(best, off);
    const int oi = __shfl_xor(bi, off);
    if (ov > best || (ov == best && oi < bi)) {
      best = ov;
      bi = oi;
    }
  }
  constexpr int NW = kArgmaxThreads / 64;
  __shared__ float sv[NW];
  __shared__ int si_[NW];
  if ((threadIdx.x & 63) == 0) {
    sv[threadIdx.x >> 6] = best;
    si_[threadIdx.x >> 6] = bi;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < NW; ++w)
      if (sv[w] > best || (sv[w] == best && si_[w] < bi)) {
        best = sv[w];
        bi = si_[w];
      }
    next[r] = bi == 0x7fffffff ? 0 : bi;
  }
}

__global__ __launch_bounds__(256) void upload16_kernel(UploadJob j) { upload_block(j, blockIdx.x); }

bool make_upload_job(const void* host_dev_ptr, void* dst, size_t bytes, uint32_t* done, uint32_t tag, UploadJob* j) {
  if (bytes % 16) return false;
  *j = UploadJob{};
  j->src = host_dev_ptr;
  j->dst = dst;
  j->n16 = (long)(bytes / 16);
  j->done = done;
  j->tag = tag;
  j->blocks = (int)std::min<long>((j->n16 + 255) / 256, kUploadMaxBlocks);
  return true;
}

int launch_upload(const UploadJob& j, hipStream_t st) {
  if (j.blocks == 0) return 0;
  hipLaunchKernelGGL(upload16_kernel, dim3(j.blocks), dim3(256), 0, st, j);
  return 0;
}

// Row-major W[N, K] -> 64x64 tiles (layout in common.h): one thread per
// destination element, zero in the padding of edge tiles. A one-time
// weight preparation; T is the element's bit pattern (2 or 4 bytes).
template <typename T>
__global__ __launch_bounds__(256) void tile_weight_kernel(const T* __restrict__ src, T* __restrict__ dst, long N,
                                                          long K, long total) {
  const long kt = (K + kWTile - 1) / kWTile;
  for (long e = (long)blockIdx.x * 256 + threadIdx.x; e < total; e += (long)gridDim.x * 256) {
    const long tile = e / kWTileElts, in = e % kWTileElts;
    const long n = (tile / kt) * kWTile + in / kWTile;
    const long k = (tile % kt) * kWTile + in % kWTile;
    dst[e] = (n < N && k < K) ? src[n * K + k] : T(0);
  }
}

int launch_tile_weight(int elt_bytes, long N, long K, const void* src, void* dst, hipStream_t st) {
  const long total = tiled_weight_elems(N, K);
  if (total == 0) return 0;
  const int blocks = (int)std::min<long>((total + 255) / 256, 8192);
  if (elt_bytes == 2)
    hipLaunchKernelGGL(tile_weight_kernel<uint16_t>, dim3(blocks), dim3(256), 0, st, (const uint16_t*)src,
                       (uint16_t*)dst, N, K, total);
  else if (elt_bytes == 4)
    hipLaunchKernelGGL(tile_weight_kernel<uint32_t>, dim3(blocks), dim3(256), 0, st, (const uint32_t*)src,
                       (uint32_t*)dst, N, K, total);
  else
    return -1;
  return 0;
}

int launch_embed(int rows, int d, int vocab, const void* table, const int32_t* tokens, void* x, hipStream_t st) {
  if (rows == 0) return 0;
  if (d % 8) return -1;
  hipLaunchKernelGGL(embed_kernel, dim3(rows), dim3(256), 0, st, (const bf16_t*)table, tokens, (bf16_t*)x, d, vocab);
  return 0;
}

int launch_gather_rows(int n, int d, const void* src, const int32_t* rows, void* dst, hipStream_t st) {
  if (n == 0) return 0;
  if (d % 8) return -1;
  hipLaunchKernelGGL(gather_rows_kernel, dim3(n), dim3(256), 0, st, (const bf16_t*)src, rows, (bf16_t*)dst, d);
  return 0;
}

int launch_argmax(int rows, int vocab, const float* logits, int32_t* next, hipStream_t st) {
  if (rows == 0) return 0;
  hipLaunchKernelGGL(argmax_kernel, dim3(rows), dim3(kArgmaxThreads), 0, st, logits, next, vocab);
  return 0;
}

}  // namespace ps
