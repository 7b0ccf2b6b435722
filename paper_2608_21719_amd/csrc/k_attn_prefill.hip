// Prefill (and chunked-prefill) causal attention over the paged KV cache,
// bf16 in, fp32 softmax, on the gfx950 matrix cores.
//
// A workgroup owns one 64-row query tile of one sequence and one KV head;
// its G waves are the G query heads of that group, so every K/V tile staged
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
#include "common.h"
#include "launch.h"

namespace ps {

namespace {
constexpr int kHd = 128;
constexpr int kQT = 64;              // query rows per workgroup
constexpr int kKT = 32;              // keys per tile (two pages)
constexpr int kKRow = kHd + 8;       // padded K row (elements)
constexpr int kVRow = kKT + 8;       // padded V^T row (elements)
}  // namespace

// Four waves = four query heads of one KV group per workgroup; groups of 8
// heads use two workgroups per KV head.
__global__ __launch_bounds__(256) void fa_prefill_kernel(const bf16_t* __restrict__ q,
                                                         const bf16_t* __restrict__ pool,
                                                         const SeqInfo* __restrict__ si,
                                                         const int32_t* __restrict__ bt,
                                                         const PrefillItem* __restrict__ items,
                                                         bf16_t* __restrict__ o, int n_kv, int G, float scale_log2) {
  constexpr int NT = 256;
  __shared__ __attribute__((aligned(16))) bf16_t sK[kKT * kKRow];
  __shared__ __attribute__((aligned(16))) bf16_t sV[kHd * kVRow];

  const int hq = G / 4;  // workgroups per KV head
  const int kvh = blockIdx.y / hq;
  const PrefillItem it = items[blockIdx.x];
  const SeqInfo s = si[it.b];
  const int n_q = n_kv * G;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int g = lane >> 5, c = lane & 31;
  const int head = kvh * G + (blockIdx.y % hq) * 4 + wave;
  const int qn = min(kQT, s.n_new - it.q_begin);       // valid rows in this tile
  const int qpos0 = s.kv_before + it.q_begin;           // position of tile row 0
  const int n_keys = qpos0 + qn;                        // keys 0 .. last query position
  const int32_t* btr = bt + s.bt_off;

  // Q^T operand: lane (g, c) holds Q[row 32cb + c][16kk + 8g .. +8]
  bf16x8_t qf[2][8];
#pragma unroll
  for (int cb = 0; cb < 2; ++cb) {
    int r = min(32 * cb + c, qn - 1);
    const bf16_t* qp = q + ((long)(s.row_start + it.q_begin + r) * n_q + head) * kHd + 8 * g;
#pragma unroll
    for (int kk = 0; kk < 8; ++kk) qf[cb][kk] = __builtin_bit_cast(bf16x8_t, *(const uint4*)(qp + 16 * kk));
  }

  f32x16_t oacc[2][4];
#pragma unroll
  for (int cb = 0; cb < 2; ++cb)
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) oacc[cb][db][r] = 0.f;
  float m[2] = {-INFINITY, -INFINITY}, l[2] = {0.f, 0.f};

  const int n_tiles = (n_keys + kKT - 1) / kKT;
  const int kv_valid = s.kv_before + s.n_new;
  for (int kt = 0; kt < n_tiles; ++kt) {
    const int k0 = kt * kKT;
    // ---- stage K [32][128] and V^T [128][32] (keys permuted per page as
    // 0-3, 8-11, 4-7, 12-15) into LDS
    for (int e = threadIdx.x; e < kKT * (kHd / 8); e += NT) {
      const int key = e >> 4, ch = e & 15;
      const int pg = (k0 + key) / kPageTokens;
      uint4 w = make_uint4(0, 0, 0, 0);
      if (k0 + key < kv_valid) {
        const bf16_t* src = pool + ((long)btr[pg] * n_kv + kvh) * (2L * kPageTokens * kHd) +
                            (long)((k0 + key) % kPageTokens) * kHd + ch * 8;
        w = *(const uint4*)src;
      }
      *(uint4*)(sK + key * kKRow + ch * 8) = w;
    }
    for (int e = threadIdx.x; e < 2 * kHd * 2; e += NT) {
      // (page in tile, dim, 16-byte half of its 16-key row)
      const int pt = e / (kHd * 2), rem = e - pt * (kHd * 2);
      const int dim = rem >> 1, hf = rem & 1;
      const int pfirst = k0 + pt * kPageTokens;  // first key of this page
      uint4 w = make_uint4(0, 0, 0, 0);
      if (pfirst < kv_valid) {
        const bf16_t* src = pool + ((long)btr[pfirst / kPageTokens] * n_kv + kvh) * (2L * kPageTokens * kHd) +
                            (long)kPageTokens * kHd + (long)dim * kPageTokens + hf * 8;
        w = *(const uint4*)src;
        // zero values of keys beyond the written length (stale memory)
        const int valid = kv_valid - pfirst - hf * 8;  // keys valid in this half
        if (valid < 8) {
          uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
          for (int i = 0; i < 8; ++i)
            if (i >= valid) ws[i >> 1] &= (i & 1) ? 0x0000ffffu : 0xffff0000u;
          w = make_uint4(ws[0], ws[1], ws[2], ws[3]);
        }
      }
      // half hf holds keys 8hf..8hf+7 = (8hf..+3, 8hf+4..+7); stored order
      // per page is [0-3][8-11][4-7][12-15] (8-byte groups)
      bf16_t* dst = sV + dim * kVRow + pt * kPageTokens;
      *(uint2*)(dst + hf * 4) = make_uint2(w.x, w.y);      // keys 8hf+0..3 -> group hf
      *(uint2*)(dst + 8 + hf * 4) = make_uint2(w.z, w.w);  // keys 8hf+4..7 -> group 2+hf
    }
    __syncthreads();

#pragma unroll
    for (int cb = 0; cb < 2; ++cb) {
      if (32 * cb >= qn) break;
      f32x16_t sacc;
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[r] = 0.f;
#pragma unroll
      for (int kk = 0; kk < 8; ++kk) {
        bf16x8_t a = __builtin_bit_cast(bf16x8_t, *(const uint4*)(sK + c * kKRow + 16 * kk + 8 * g));
        sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[cb][kk], sacc, 0, 0, 0);
      }
      // sacc[r] = score(key 8(r/4) + 4g + r%4, query c)
      const int qpos = qpos0 + 32 * cb + c;
      float mx = -INFINITY;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = k0 + 8 * (r >> 2) + 4 * g + (r & 3);
        sacc[r] = (key <= qpos) ? sacc[r] * scale_log2 : -INFINITY;
        mx = fmaxf(mx, sacc[r]);
      }
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m[cb], mx);
      const float alpha = (m_new == -INFINITY) ? 1.f : exp2f(m[cb] - m_new);
      uint32_t pk[8];
      float psum = 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        float p0 = (m_new == -INFINITY) ? 0.f : exp2f(sacc[2 * i] - m_new);
        float p1 = (m_new == -INFINITY) ? 0.f : exp2f(sacc[2 * i + 1] - m_new);
        pk[i] = pack_bf2(p0, p1);
        psum += bf_lo(pk[i]) + bf_hi(pk[i]);
      }
      l[cb] = l[cb] * alpha + psum;
      m[cb] = m_new;
#pragma unroll
      for (int db = 0; db < 4; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[cb][db][r] *= alpha;
#pragma unroll
      for (int kk2 = 0; kk2 < 2; ++kk2) {
        const bf16x8_t bp =
            __builtin_bit_cast(bf16x8_t, make_uint4(pk[4 * kk2], pk[4 * kk2 + 1], pk[4 * kk2 + 2], pk[4 * kk2 + 3]));
#pragma unroll
        for (int db = 0; db < 4; ++db) {
          bf16x8_t a = __builtin_bit_cast(
              bf16x8_t, *(const uint4*)(sV + (32 * db + c) * kVRow + kk2 * kPageTokens + 8 * g));
          oacc[cb][db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, bp, oacc[cb][db], 0, 0, 0);
        }
      }
    }
    __syncthreads();
  }

  // ---- normalise and store: lane holds query c, dims 32db + 8(r/4) + 4g + r%4
#pragma unroll
  for (int cb = 0; cb < 2; ++cb) {
    const int r0 = 32 * cb + c;
    if (r0 >= qn) continue;
    const float L = l[cb] + __shfl_xor(l[cb], 32);
    const float inv = 1.f / L;
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
