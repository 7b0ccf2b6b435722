// Shared device/host definitions for the gfx950 kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ps {

typedef uint16_t bf16_t;  // raw bfloat16 bits

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(short)))) short s16x4_t;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int kPageTokens = 16;
constexpr int kGateUpBlock = 32;
constexpr long kMaxDecodeItems = 65535;  // decode attention work items per launch (grid y)
// Linear weights W[N, K] are stored in 64x64 tiles (tile (i, j) at index
// i * ceil(K/64) + j, row-major inside; edge tiles zero-padded).
constexpr int kWTile = 64;
constexpr int kWTileElts = kWTile * kWTile;
__host__ __device__ inline long tiled_weight_elems(long N, long K) {
  return ((N + kWTile - 1) / kWTile) * ((K + kWTile - 1) / kWTile) * kWTileElts;
}
__host__ __device__ inline long tiled_index(long n, long k, long K) {
  const long kt = (K + kWTile - 1) / kWTile;
  return ((n / kWTile) * kt + k / kWTile) * kWTileElts + (n % kWTile) * kWTile + (k % kWTile);
}

__device__ __forceinline__ float bf2f(bf16_t b) { return __uint_as_float(((uint32_t)b) << 16); }
__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2_t;

// float -> bf16 bits, round to nearest even: the float->__bf16 conversion
// lowers to gfx950's v_cvt_pk_bf16_f32 (RNE, NaN stays NaN).
__device__ __forceinline__ bf16_t f2bf(float f) { return __builtin_bit_cast(bf16_t, (__bf16)f); }
__device__ __forceinline__ uint32_t pack_bf2(float lo, float hi) {
  bf16x2_t v;
  v[0] = (__bf16)lo;
  v[1] = (__bf16)hi;
  return __builtin_bit_cast(uint32_t, v);
}

template <typename T> struct Elt;
template <> struct Elt<float> {
  __device__ static float load(const float* p, long i) { return p[i]; }
  __device__ static void store(float* p, long i, float v) { p[i] = v; }
};
template <> struct Elt<bf16_t> {
  __device__ static float load(const bf16_t* p, long i) { return bf2f(p[i]); }
  __device__ static void store(bf16_t* p, long i, float v) { p[i] = f2bf(v); }
};

// Per-call sequence record uploaded with the call's metadata.
struct SeqInfo {
  int32_t kv_before;  // committed length before this call (first new position)
  int32_t n_new;      // rows this call adds for the sequence
  int32_t row_start;  // first row of the sequence in the call's activations
  int32_t bt_off;     // offset of its block-table row in the compact table
};

// One split of decode attention: logical pages [page_begin, page_end) of
// batch entry b; part is the index of its partial result.
struct DecodeItem {
  int32_t b;
  int32_t page_begin;
  int32_t page_end;
  int32_t part;
};

// One query tile of prefill attention.
struct PrefillItem {
  int32_t b;
  int32_t q_begin;  // first new row of the tile, relative to the sequence's new rows
};

}  // namespace ps
