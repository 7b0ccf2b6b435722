// Decode attention over the paged KV cache (gfx950).
//
// Split-K: a work item is (batch entry, logical page range, kv head). Its
// four waves walk the range's 16-token pages in logical order (wave w takes
// pages w, w+4, ...), so the arithmetic never depends on where pages sit
// physically. Per page a wave reads the 4 KiB key block with 16-byte loads
// and the 4 KiB V^T block with 8-byte loads, non-temporal (KV is streamed
// once per step), keeping kPrefetch pages in flight beyond the one it works
// on; the block table is read with scalar loads, so fetching the next page
// id never waits on the vector loads already in flight. The kv head is the
// fastest grid index: workgroups running together read the adjacent heads
// of the same pages. A launch may cap its workgroups (the mixed step does,
// to leave compute units to the GEMMs beside it); each then walks items
// y, y + gridDim.y, ... in turn. Each page does all of the group's query heads at once
// on the matrix cores:
//
//   S^T[tok, head] = K[tok, :] . q[head, :]     4 x v_mfma_f32_16x16x32_bf16
//   O[head, dim]  += P[head, tok] V[tok, dim]   8 x v_mfma_f32_16x16x16_bf16
//
// The 16-row MFMA tile holds the G (<= 16) heads of one KV group; rows
// beyond G are padding. The S^T output layout (lane = head, 4 tokens per
// lane) is exactly the A-operand layout P needs, so no shuffle sits between
// the two products. Online softmax runs in base 2 on fp32 scores; P is
// rounded to bf16 for the PV product and the normaliser sums those same
// rounded values (so V == 1 gives exactly 1). The pass is bound by HBM:
// 4 FLOP per KV byte.
//
// A second kernel merges the splits of each (sequence, head) in split order
// (log-sum-exp), which keeps the result deterministic.
#include "common.h"
#include "launch.h"

namespace ps {

constexpr int kHd = 128;      // head_dim of the MFMA path
constexpr int kPrefetch = 2;  // pages in flight per wave beyond the current one

typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

template <int G>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void decode_attn_kernel(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ pool, const SeqInfo* __restrict__ si,
    const int32_t* __restrict__ bt, const DecodeItem* __restrict__ items, float* __restrict__ part_o,
    float* __restrict__ part_ml, int n_kv, int n_items, float scale_log2) {
  static_assert(G <= 16, "one 16-row MFMA tile per KV group");
  constexpr int D = kPrefetch;
  const int kvh = blockIdx.x;
  // items blockIdx.y, + gridDim.y, ...: one each when the grid covers them
  // all, several when the launch caps its workgroups
  for (int iy = blockIdx.y; iy < n_items; iy += gridDim.y) {
  const DecodeItem it = items[iy];
  const SeqInfo s = si[it.b];
  const int kv_len = s.kv_before + s.n_new;
  const int n_q = n_kv * G;
  // wave index made wave-uniform so page ids and page addresses stay scalar
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4, c = lane & 15;

  // Q operand (B of the S^T product): lane holds q[head c][32j + 8g .. +8].
  bf16x8_t qb[4];
  {
    const bf16_t* qp = q + ((long)it.b * n_q + kvh * G + (c < G ? c : 0)) * kHd + 8 * g;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      uint4 w = (c < G) ? *(const uint4*)(qp + 32 * j) : make_uint4(0, 0, 0, 0);
      qb[j] = __builtin_bit_cast(bf16x8_t, w);
    }
  }

  float m = -INFINITY, l = 0.f;
  f32x4_t acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const int32_t* btr = bt + s.bt_off;
  const int last_page = (kv_len - 1) / kPageTokens;
  const int koff = c * kHd + 8 * g;                               // + 32 j
  const int voff = kPageTokens * kHd + c * kPageTokens + 4 * g;   // + 16 blk kPageTokens
  const long head_off = (long)kvh * (2L * kPageTokens * kHd);
  const long page_stride = (long)n_kv * (2L * kPageTokens * kHd);

  // three static register sets form the page ring (two pages in flight while
  // one is consumed); a ring indexed at run time would be copied through
  // registers, and each copy of an in-flight load waits for it
  static_assert(kPrefetch == 2, "the page ring below is unrolled for two pages in flight");
  struct PageRegs {
    uint4 k[4];
    uint2 v[8];
  };
  PageRegs r0, r1, r2;
  auto load_page = [&](int p, PageRegs& r) {
    const bf16_t* base = pool + (long)btr[p] * page_stride + head_off;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      r.k[j] = __builtin_bit_cast(uint4, __builtin_nontemporal_load((const u32x4_t*)(base + koff + 32 * j)));
#pragma unroll
    for (int blk = 0; blk < 8; ++blk)
      r.v[blk] = __builtin_bit_cast(
          uint2, __builtin_nontemporal_load((const u32x2_t*)(base + voff + 16 * blk * kPageTokens)));
  };

  // consume one page held in `cur`
  auto page_compute = [&](int p, PageRegs& cur) {
    // tokens past the written length (last page only) hold stale memory:
    // zero their V so 0 * garbage cannot produce NaN (branch-free, so no
    // wait on the page's loads is placed on a path of its own)
    const int valid = (p == last_page) ? kv_len - p * kPageTokens : kPageTokens;  // 1..16
    const uint32_t m0 = (4 * g + 0 < valid ? 0x0000ffffu : 0u) | (4 * g + 1 < valid ? 0xffff0000u : 0u);
    const uint32_t m1 = (4 * g + 2 < valid ? 0x0000ffffu : 0u) | (4 * g + 3 < valid ? 0xffff0000u : 0u);
#pragma unroll
    for (int blk = 0; blk < 8; ++blk) cur.v[blk] = make_uint2(cur.v[blk].x & m0, cur.v[blk].y & m1);

    f32x4_t st = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < 4; ++j)
      st = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, cur.k[j]), qb[j], st, 0, 0, 0);
    // st[r] = score(token 4g + r, head c)
    float sc[4];
    float mx = -INFINITY;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int tok = p * kPageTokens + 4 * g + r;
      sc[r] = (tok < kv_len) ? st[r] * scale_log2 : -INFINITY;
      mx = fmaxf(mx, sc[r]);
    }
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m, mx);
    const float alpha = exp2f(m - m_new);
    float pr[4];
    uint32_t pk[2];
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      pk[r] = pack_bf2(exp2f(sc[2 * r] - m_new), exp2f(sc[2 * r + 1] - m_new));
      pr[2 * r] = bf_lo(pk[r]);
      pr[2 * r + 1] = bf_hi(pk[r]);
    }
    l = l * alpha + (pr[0] + pr[1] + pr[2] + pr[3]);
    m = m_new;
    // acc rows are heads 4g + r: fetch their rescale factors
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float a_r = __shfl(alpha, 4 * g + r);
#pragma unroll
      for (int blk = 0; blk < 8; ++blk) acc[blk][r] *= a_r;
    }
    const s16x4_t pa = __builtin_bit_cast(s16x4_t, make_uint2(pk[0], pk[1]));
#pragma unroll
    for (int blk = 0; blk < 8; ++blk)
      acc[blk] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(pa, __builtin_bit_cast(s16x4_t, cur.v[blk]), acc[blk],
                                                           0, 0, 0);
  };

  // wave pages p0, p0 + 4, ...: r0 holds page p and r1 page p + 4 at the top
  // of every round; a round consumes three pages and requests three
  const int end = it.page_end;
  int p = it.page_begin + wave;
  if (p < end) load_page(p, r0);
  __builtin_amdgcn_sched_barrier(0);  // page p's loads first (the wait for it below counts on that order)
  if (p + 4 < end) load_page(p + 4, r1);
  __builtin_amdgcn_sched_barrier(0);
  // The scheduling barriers keep the order below: left free, the scheduler
  // hoists the next page's score MFMAs above this page's, so every round
  // began by waiting for both pages in flight (vmcnt(0)) and issued its
  // next request only after that.
  for (; p + 16 < end; p += 12) {  // steady state: every request is a real page
    load_page(p + 8, r2);
    __builtin_amdgcn_sched_barrier(0);
    page_compute(p, r0);
    __builtin_amdgcn_sched_barrier(0);
    load_page(p + 12, r0);
    __builtin_amdgcn_sched_barrier(0);
    page_compute(p + 4, r1);
    __builtin_amdgcn_sched_barrier(0);
    load_page(p + 16, r1);
    __builtin_amdgcn_sched_barrier(0);
    page_compute(p + 8, r2);
    __builtin_amdgcn_sched_barrier(0);
  }
  if (p < end) {  // at most four pages left: p, p + 4, p + 8, p + 12
    if (p + 8 < end) load_page(p + 8, r2);
    page_compute(p, r0);
    if (p + 4 < end) {
      if (p + 12 < end) load_page(p + 12, r0);
      page_compute(p + 4, r1);
      if (p + 8 < end) {
        page_compute(p + 8, r2);
        if (p + 12 < end) page_compute(p + 12, r0);
      }
    }
  }
  // per-head normaliser: sum the four lane groups
  l += __shfl_xor(l, 16);
  l += __shfl_xor(l, 32);

  // merge the four waves through LDS
  __shared__ float s_acc[4][G][kHd];
  __shared__ float s_m[4][16], s_l[4][16];
  if (lane < 16) {
    s_m[wave][lane] = m;
    s_l[wave][lane] = l;
  }
#pragma unroll
  for (int blk = 0; blk < 8; ++blk)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int head = 4 * g + r;
      if (head < G) s_acc[wave][head][16 * blk + c] = acc[blk][r];
    }
  __syncthreads();
  const long part = (long)it.part * n_kv + kvh;
  for (int e = threadIdx.x; e < G * kHd; e += 256) {
    const int head = e / kHd, dim = e - head * kHd;
    float M = fmaxf(fmaxf(s_m[0][head], s_m[1][head]), fmaxf(s_m[2][head], s_m[3][head]));
    float o = 0.f, L = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float f = (s_m[w][head] == -INFINITY) ? 0.f : exp2f(s_m[w][head] - M);
      o += s_acc[w][head][dim] * f;
      L += s_l[w][head] * f;
    }
    part_o[(part * G + head) * kHd + dim] = o;
    if (dim == 0) {
      part_ml[(part * G + head) * 2 + 0] = M;
      part_ml[(part * G + head) * 2 + 1] = L;
    }
  }
  __syncthreads();  // the next item reuses s_acc, s_m, s_l
  }
}

// o[b, head, :] = sum_s o_s 2^(m_s - M) / sum_s l_s 2^(m_s - M), splits in order.
__global__ __launch_bounds__(128) void decode_combine_kernel(const float* __restrict__ part_o,
                                                             const float* __restrict__ part_ml,
                                                             const int32_t* __restrict__ part_begin,
                                                             const int32_t* __restrict__ part_count,
                                                             bf16_t* __restrict__ o, int n_kv, int G) {
  const int b = blockIdx.x, head = blockIdx.y, dim = threadIdx.x;
  const int kvh = head / G, hg = head - kvh * G;
  const int p0 = part_begin[b], np = part_count[b];
  const long stride = (long)n_kv * G;  // between consecutive splits of one (sequence, head)
  const long pi0 = ((long)p0 * n_kv + kvh) * G + hg;
  // Loads go four splits at a time so that their latencies overlap; the
  // arithmetic is the same sequence in split order as one split at a time.
  float M = -INFINITY;
  int i = 0;
  for (; i + 4 <= np; i += 4) {
    float mm[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) mm[u] = part_ml[(pi0 + (i + u) * stride) * 2];
#pragma unroll
    for (int u = 0; u < 4; ++u) M = fmaxf(M, mm[u]);
  }
  for (; i < np; ++i) M = fmaxf(M, part_ml[(pi0 + i * stride) * 2]);
  float acc = 0.f, L = 0.f;
  i = 0;
  for (; i + 4 <= np; i += 4) {
    float ov[4], mv[4], lv[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const long pi = pi0 + (i + u) * stride;
      ov[u] = part_o[pi * kHd + dim];
      mv[u] = part_ml[pi * 2];
      lv[u] = part_ml[pi * 2 + 1];
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const float f = exp2f(mv[u] - M);
      acc += ov[u] * f;
      L += lv[u] * f;
    }
  }
  for (; i < np; ++i) {
    const long pi = pi0 + i * stride;
    const float f = exp2f(part_ml[pi * 2] - M);
    acc += part_o[pi * kHd + dim] * f;
    L += part_ml[pi * 2 + 1] * f;
  }
  o[((long)b * n_kv * G + head) * kHd + dim] = f2bf(acc / L);
}

int launch_decode_attn(int G, int n_items, int n_kv, int n_seqs, const void* q, const void* pool_layer,
                       const SeqInfo* si, const int32_t* bt, const DecodeItem* items, float* part_o,
                       float* part_ml, const int32_t* part_begin, const int32_t* part_count, void* o,
                       float scale_log2, hipStream_t st, int max_wg) {
  if (n_seqs == 0) return 0;
  if (n_items > kMaxDecodeItems) return -1;
  int gy = n_items;
  if (max_wg > 0) gy = std::max(1, std::min(n_items, max_wg / n_kv));
  dim3 grid(n_kv, gy);
  switch (G) {
    case 1: hipLaunchKernelGGL(decode_attn_kernel<1>, grid, dim3(256), 0, st, (const bf16_t*)q, (const bf16_t*)pool_layer, si, bt, items, part_o, part_ml, n_kv, n_items, scale_log2); break;
    case 2: hipLaunchKernelGGL(decode_attn_kernel<2>, grid, dim3(256), 0, st, (const bf16_t*)q, (const bf16_t*)pool_layer, si, bt, items, part_o, part_ml, n_kv, n_items, scale_log2); break;
    case 4: hipLaunchKernelGGL(decode_attn_kernel<4>, grid, dim3(256), 0, st, (const bf16_t*)q, (const bf16_t*)pool_layer, si, bt, items, part_o, part_ml, n_kv, n_items, scale_log2); break;
    case 8: hipLaunchKernelGGL(decode_attn_kernel<8>, grid, dim3(256), 0, st, (const bf16_t*)q, (const bf16_t*)pool_layer, si, bt, items, part_o, part_ml, n_kv, n_items, scale_log2); break;
    case 16: hipLaunchKernelGGL(decode_attn_kernel<16>, grid, dim3(256), 0, st, (const bf16_t*)q, (const bf16_t*)pool_layer, si, bt, items, part_o, part_ml, n_kv, n_items, scale_log2); break;
    default: return -1;
  }
  hipLaunchKernelGGL(decode_combine_kernel, dim3(n_seqs, n_kv * G), dim3(kHd), 0, st, part_o, part_ml,
                     part_begin, part_count, (bf16_t*)o, n_kv, G);
  return 0;
}

// ---------------------------------------------------------------- generic
// Vector-ALU attention for fp32 layers (and any head_dim <= 128): one wave
// per (row, query head), keys 0..pos of the row's sequence walked in order
// with an online softmax in fp32.
template <typename T>
__global__ __launch_bounds__(64) void attn_generic_kernel(const T* __restrict__ q, const T* __restrict__ pool,
                                                          const SeqInfo* __restrict__ si,
                                                          const int32_t* __restrict__ bt, T* __restrict__ o,
                                                          int row0, int n_seqs, int n_q, int n_kv, int hd,
                                                          float scale) {
  const int row = row0 + blockIdx.x, head = blockIdx.y, lane = threadIdx.x;
  int lo = 0, hi = n_seqs - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (si[mid].row_start <= row) lo = mid; else hi = mid - 1;
  }
  const SeqInfo s = si[lo];
  const int pos = s.kv_before + (row - s.row_start);
  const int kvh = head / (n_q / n_kv);
  float qv[2], acc[2] = {0.f, 0.f};
  for (int e = 0; e < 2; ++e) {
    int dim = lane + 64 * e;
    qv[e] = dim < hd ? Elt<T>::load(q, ((long)row * n_q + head) * hd + dim) : 0.f;
  }
  float m = -INFINITY, l = 0.f;
  for (int j = 0; j <= pos; ++j) {
    const long base = ((long)bt[s.bt_off + j / kPageTokens] * n_kv + kvh) * (2L * kPageTokens * hd);
    const int slot = j % kPageTokens;
    float part = 0.f, vv[2] = {0.f, 0.f};
    for (int e = 0; e < 2; ++e) {
      int dim = lane + 64 * e;
      if (dim < hd) {
        part += qv[e] * Elt<T>::load(pool, base + (long)slot * hd + dim);
        vv[e] = Elt<T>::load(pool, base + (long)kPageTokens * hd + (long)dim * kPageTokens + slot);
      }
    }
    for (int off = 32; off > 0; off >>= 1) part += __shfl_xor(part, off);
    const float sc = part * scale;
    const float m_new = fmaxf(m, sc);
    const float a = expf(m - m_new), p = expf(sc - m_new);
    l = l * a + p;
    for (int e = 0; e < 2; ++e) acc[e] = acc[e] * a + p * vv[e];
    m = m_new;
  }
  for (int e = 0; e < 2; ++e) {
    int dim = lane + 64 * e;
    if (dim < hd) Elt<T>::store(o, ((long)row * n_q + head) * hd + dim, acc[e] / l);
  }
}

int launch_attn_generic(int dt, int row0, int rows, int n_seqs, int n_q, int n_kv, int hd, const void* q,
                        const void* pool_layer, const SeqInfo* si, const int32_t* bt, void* o, float scale,
                        hipStream_t st) {
  if (rows == 0) return 0;
  if (hd > 128) return -1;
  dim3 grid(rows, n_q);
  if (dt == 1)
    hipLaunchKernelGGL(attn_generic_kernel<bf16_t>, grid, dim3(64), 0, st, (const bf16_t*)q,
                       (const bf16_t*)pool_layer, si, bt, (bf16_t*)o, row0, n_seqs, n_q, n_kv, hd, scale);
  else
    hipLaunchKernelGGL(attn_generic_kernel<float>, grid, dim3(64), 0, st, (const float*)q,
                       (const float*)pool_layer, si, bt, (float*)o, row0, n_seqs, n_q, n_kv, hd, scale);
  return 0;
}

}  // namespace ps
