// Attainable ceilings of one MI355X (gfx950), measured rather than taken
// from the data sheet: HBM streaming read and copy bandwidth, the dense
// bf16 MFMA rate of v_mfma_f32_32x32x16_bf16 on register operands (near
// constant, and random bits changing every product, as a GEMM on real data
// sees; also v_mfma_f32_16x16x32_bf16 on the same random data), and
// whether MFMA and vector-ALU work issued on the same SIMD overlap in time.
// `ceilings mfma-random [seconds [32x32x16|16x16x32]]` runs only the
// random-operand rates (or one of them) for about as long as asked, so that
// clock and power can be sampled beside it.
// A standalone program (not part of libps); every buffer is allocated here
// and every kernel indexes inside it.
#include <hip/hip_runtime.h>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#define CHECK(x)                                                                 \
  do {                                                                           \
    hipError_t e_ = (x);                                                         \
    if (e_ != hipSuccess) {                                                      \
      std::fprintf(stderr, "%s failed: %s\n", #x, hipGetErrorString(e_));       \
      std::exit(1);                                                              \
    }                                                                            \
  } while (0)

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Random bf16 operands that change from one product to the next: each wave
// holds 4 A and 4 B fragments of random sign and mantissa bits (exponent
// 126 or 127, so every value is normal and no sum overflows) and pairs
// A j with B (j + r) % 4 in rotation r. SHAPE 0: 16 v_mfma_f32_32x32x16_bf16
// per trip over 4 accumulators; SHAPE 1: 32 v_mfma_f32_16x16x32_bf16 (the
// same FLOPs) over 16, each reused every 16 products. One trip is 524288
// FLOP per wave.
template <int SHAPE>
__global__ __launch_bounds__(256) void mfma_random(float* out, int trips) {
  unsigned h = (blockIdx.x * 256u + threadIdx.x) * 0x9E3779B9u + 0x7F4A7C15u;
  auto next = [&]() {
    h ^= h << 13;
    h ^= h >> 17;
    h ^= h << 5;
    return h;
  };
  auto rnd_bf16 = [&]() {
    const unsigned x = next();
    const unsigned short bits = (unsigned short)((x & 0x807Fu) | ((x >> 8) & 1u ? 0x3F80u : 0x3F00u));
    return __builtin_bit_cast(__bf16, bits);
  };
  bf16x8 a[4], b[4];
  for (int j = 0; j < 4; ++j)
    for (int e = 0; e < 8; ++e) {
      a[j][e] = rnd_bf16();
      b[j][e] = rnd_bf16();
    }
  float s = 0.f;
  if constexpr (SHAPE == 0) {
    f32x16 acc[4];
    for (int j = 0; j < 4; ++j)
      for (int r = 0; r < 16; ++r) acc[j][r] = 0.f;
    for (int t = 0; t < trips; ++t) {
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[j], b[(j + r) & 3], acc[j], 0, 0, 0);
    }
    for (int j = 0; j < 4; ++j)
      for (int r = 0; r < 16; ++r) s += acc[j][r];
  } else {
    f32x4 acc[16];
    for (int j = 0; j < 16; ++j)
      for (int r = 0; r < 4; ++r) acc[j][r] = 0.f;
    for (int t = 0; t < trips; ++t) {
#pragma unroll
      for (int r = 0; r < 2; ++r)
#pragma unroll
        for (int j = 0; j < 16; ++j)
          acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[j & 3], b[((j >> 2) + r) & 3], acc[j], 0, 0, 0);
    }
    for (int j = 0; j < 16; ++j)
      for (int r = 0; r < 4; ++r) s += acc[j][r];
  }
  out[blockIdx.x * 256 + threadIdx.x] = s;
}

// grid-stride non-temporal 16-byte reads, folded so the loads stay live
__global__ void hbm_read(const u32x4* __restrict__ p, long n, unsigned* out) {
  u32x4 acc = {0, 0, 0, 0};
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (long)gridDim.x * blockDim.x)
    acc ^= __builtin_nontemporal_load(p + i);
  if ((acc.x ^ acc.y ^ acc.z ^ acc.w) == 0x9e3779b9u) out[0] = 1;
}

__global__ void hbm_copy(const u32x4* __restrict__ p, u32x4* __restrict__ q, long n) {
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (long)gridDim.x * blockDim.x) q[i] = p[i];
}

// MODE 0: MFMA only; 1: vector FMAs only; 2: both in every wave (accumulators
// in VGPRs); 3: both, accumulators held in AGPRs. Four independent 32x32
// accumulators and four independent FMA chains per wave.
template <int MODE>
__global__ __launch_bounds__(256) void issue_mix(float* out, int iters) {
  f32x16 acc[4];
  for (int j = 0; j < 4; ++j)
    for (int r = 0; r < 16; ++r) acc[j][r] = 0.f;
  bf16x8 a, b;
  for (int e = 0; e < 8; ++e) {
    a[e] = (__bf16)(1e-3f * (float)(threadIdx.x + e));
    b[e] = (__bf16)(2e-3f * (float)e);
  }
  float v0 = threadIdx.x * 1e-3f, v1 = v0 + 1.f, v2 = v0 + 2.f, v3 = v0 + 3.f;
  for (int i = 0; i < iters; ++i) {
    if (MODE != 1) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[j], 0, 0, 0);
        if (MODE == 3) asm volatile("" : "+a"(acc[j]));
      }
    }
    if (MODE != 0) {
#pragma unroll
      for (int k = 0; k < 16; ++k) {
        v0 = fmaf(v0, 1.0001f, 0.5f);
        v1 = fmaf(v1, 0.9999f, 0.25f);
        v2 = fmaf(v2, 1.0002f, 0.125f);
        v3 = fmaf(v3, 0.9998f, 0.0625f);
      }
    }
  }
  float s = v0 + v1 + v2 + v3;
  for (int j = 0; j < 4; ++j)
    for (int r = 0; r < 16; ++r) s += acc[j][r];
  out[(long)blockIdx.x * blockDim.x + threadIdx.x] = s;
}

// Workgroups of eight waves, one per CU: waves w and w + 4 share SIMD w % 4.
// MODE 0: waves 0-3 run MFMAs, waves 4-7 nothing; 1: waves 0-3 nothing,
// waves 4-7 vector FMA chains; 2: both, on different waves of one SIMD.
template <int MODE>
__global__ __launch_bounds__(512) void cross_wave(float* out, int iters) {
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const bool do_m = wave < 4 && MODE != 1, do_v = wave >= 4 && MODE != 0;
  f32x16 acc[4];
  for (int j = 0; j < 4; ++j)
    for (int r = 0; r < 16; ++r) acc[j][r] = 0.f;
  bf16x8 a, b;
  for (int e = 0; e < 8; ++e) {
    a[e] = (__bf16)(1e-3f * (float)(threadIdx.x + e));
    b[e] = (__bf16)(2e-3f * (float)e);
  }
  float v0 = threadIdx.x * 1e-3f, v1 = v0 + 1.f, v2 = v0 + 2.f, v3 = v0 + 3.f;
  for (int i = 0; i < iters; ++i) {
    if (do_m) {
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[j], 0, 0, 0);
    }
    if (do_v) {
#pragma unroll
      for (int k = 0; k < 16; ++k) {
        v0 = fmaf(v0, 1.0001f, 0.5f);
        v1 = fmaf(v1, 0.9999f, 0.25f);
        v2 = fmaf(v2, 1.0002f, 0.125f);
        v3 = fmaf(v3, 0.9998f, 0.0625f);
      }
    }
  }
  float s = v0 + v1 + v2 + v3;
  for (int j = 0; j < 4; ++j)
    for (int r = 0; r < 16; ++r) s += acc[j][r];
  out[(long)blockIdx.x * blockDim.x + threadIdx.x] = s;
}

// Eight waves per CU (two per SIMD), every wave running 4 MFMAs and 64 FMAs
// (four chains) per iteration, enough to keep the vector ALU busy; the waves
// 4-7 first run OFF extra FMAs, so the two waves of a SIMD start out of phase.
template <int OFF>
__global__ __launch_bounds__(512) void phase_mix(float* out, int iters) {
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  f32x16 acc[4];
  for (int j = 0; j < 4; ++j)
    for (int r = 0; r < 16; ++r) acc[j][r] = 0.f;
  bf16x8 a, b;
  for (int e = 0; e < 8; ++e) {
    a[e] = (__bf16)(1e-3f * (float)(threadIdx.x + e));
    b[e] = (__bf16)(2e-3f * (float)e);
  }
  float v0 = threadIdx.x * 1e-3f, v1 = v0 + 1.f, v2 = v0 + 2.f, v3 = v0 + 3.f;
  if (wave >= 4)
    for (int k = 0; k < OFF / 4; ++k) {
      v0 = fmaf(v0, 1.0001f, 0.5f);
      v1 = fmaf(v1, 0.9999f, 0.25f);
      v2 = fmaf(v2, 1.0002f, 0.125f);
      v3 = fmaf(v3, 0.9998f, 0.0625f);
    }
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[j], 0, 0, 0);
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      v0 = fmaf(v0, 1.0001f, 0.5f);
      v1 = fmaf(v1, 0.9999f, 0.25f);
      v2 = fmaf(v2, 1.0002f, 0.125f);
      v3 = fmaf(v3, 0.9998f, 0.0625f);
    }
  }
  float s = v0 + v1 + v2 + v3;
  for (int j = 0; j < 4; ++j)
    for (int r = 0; r < 16; ++r) s += acc[j][r];
  out[(long)blockIdx.x * blockDim.x + threadIdx.x] = s;
}

static float time_ms(hipEvent_t e0, hipEvent_t e1) {
  float ms = 0.f;
  CHECK(hipEventElapsedTime(&ms, e0, e1));
  return ms;
}

// bf16 MFMA rate on random operands, one 4-wave workgroup per CU (one wave
// per SIMD, as the tile GEMM runs), each shape timed over about `seconds`
static void mfma_random_rates(int cus, double seconds, hipEvent_t e0, hipEvent_t e1, int only_shape = -1) {
  float* out = nullptr;
  CHECK(hipMalloc(&out, (size_t)cus * 256 * sizeof(float)));
  for (int shape = 0; shape < 2; ++shape) {
    if (only_shape >= 0 && shape != only_shape) continue;
    auto launch = [&](int trips) {
      if (shape == 0) hipLaunchKernelGGL(mfma_random<0>, dim3(cus), dim3(256), 0, 0, out, trips);
      else hipLaunchKernelGGL(mfma_random<1>, dim3(cus), dim3(256), 0, 0, out, trips);
    };
    // size a launch to about 50 ms from a short one, then repeat it
    const int probe_trips = 20000;
    launch(probe_trips);
    CHECK(hipEventRecord(e0));
    launch(probe_trips);
    CHECK(hipEventRecord(e1));
    CHECK(hipEventSynchronize(e1));
    float ms0 = 0.f;
    CHECK(hipEventElapsedTime(&ms0, e0, e1));
    const int trips = (int)(probe_trips * 50.0 / (ms0 > 0.01f ? ms0 : 0.01f));
    const int reps = (int)(seconds * 1000.0 / 50.0) + 1;
    CHECK(hipEventRecord(e0));
    for (int r = 0; r < reps; ++r) launch(trips);
    CHECK(hipEventRecord(e1));
    CHECK(hipEventSynchronize(e1));
    CHECK(hipGetLastError());
    float ms = 0.f;
    CHECK(hipEventElapsedTime(&ms, e0, e1));
    const double flop = (double)cus * 4 * (double)trips * reps * 524288.0;
    std::printf("mfma %s bf16, random operands changing every product: %.0f TFLOP/s (%.0f ms)\n",
                shape == 0 ? "32x32x16" : "16x16x32", flop / (ms * 1e-3) / 1e12, ms);
    std::fflush(stdout);
  }
  CHECK(hipFree(out));
}

int main(int argc, char** argv) {
  int dev = 0, cus = 0;
  CHECK(hipGetDevice(&dev));
  CHECK(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
  hipEvent_t e0, e1;
  CHECK(hipEventCreate(&e0));
  CHECK(hipEventCreate(&e1));
  if (argc > 1 && std::strcmp(argv[1], "mfma-random") == 0) {
    const int only = argc > 3 ? (std::strcmp(argv[3], "16x16x32") == 0 ? 1 : 0) : -1;
    mfma_random_rates(cus, argc > 2 ? std::atof(argv[2]) : 1.0, e0, e1, only);
    return 0;
  }

  // ---- HBM: 4 GiB source, far beyond the caches
  const long bytes = 4L << 30, n = bytes / 16;
  u32x4 *a = nullptr, *b = nullptr;
  unsigned* flag = nullptr;
  CHECK(hipMalloc(&a, bytes));
  CHECK(hipMalloc(&b, bytes / 2));
  CHECK(hipMalloc(&flag, 4));
  CHECK(hipMemset(a, 1, bytes));
  CHECK(hipDeviceSynchronize());
  double best_rd = 0, best_cp = 0;
  for (int grid : {1024, 2048, 4096, 8192}) {
    hipLaunchKernelGGL(hbm_read, dim3(grid), dim3(256), 0, 0, a, n, flag);
    CHECK(hipEventRecord(e0));
    for (int i = 0; i < 10; ++i) hipLaunchKernelGGL(hbm_read, dim3(grid), dim3(256), 0, 0, a, n, flag);
    CHECK(hipEventRecord(e1));
    CHECK(hipEventSynchronize(e1));
    const double rd = 10.0 * bytes / (time_ms(e0, e1) * 1e-3) / 1e9;
    // copy half the source into b: bytes / 2 read + bytes / 2 written
    hipLaunchKernelGGL(hbm_copy, dim3(grid), dim3(256), 0, 0, a, b, n / 2);
    CHECK(hipEventRecord(e0));
    for (int i = 0; i < 10; ++i) hipLaunchKernelGGL(hbm_copy, dim3(grid), dim3(256), 0, 0, a, b, n / 2);
    CHECK(hipEventRecord(e1));
    CHECK(hipEventSynchronize(e1));
    const double cp = 10.0 * bytes / (time_ms(e0, e1) * 1e-3) / 1e9;
    std::printf("hbm  grid %5d x 256: read %6.0f GB/s   copy %6.0f GB/s (read + write)\n", grid, rd, cp);
    best_rd = rd > best_rd ? rd : best_rd;
    best_cp = cp > best_cp ? cp : best_cp;
  }
  CHECK(hipGetLastError());
  CHECK(hipFree(a));
  CHECK(hipFree(b));
  CHECK(hipFree(flag));

  // ---- matrix cores and vector ALU: two workgroups of four waves per CU
  // (two waves per SIMD); the first timed pass follows a long warm-up so the
  // clock has settled
  const int blocks = 2 * cus, iters = 20000;
  float* out = nullptr;
  CHECK(hipMalloc(&out, (size_t)blocks * 256 * sizeof(float)));
  auto run = [&](auto kern) {
    for (int w = 0; w < 3; ++w) hipLaunchKernelGGL(kern, dim3(blocks), dim3(256), 0, 0, out, iters);
    CHECK(hipEventRecord(e0));
    hipLaunchKernelGGL(kern, dim3(blocks), dim3(256), 0, 0, out, iters);
    CHECK(hipEventRecord(e1));
    CHECK(hipEventSynchronize(e1));
    return (double)time_ms(e0, e1);
  };
  const double t_m = run(issue_mix<0>), t_v = run(issue_mix<1>), t_b = run(issue_mix<2>), t_a = run(issue_mix<3>);
  CHECK(hipGetLastError());
  const double mfma_flop = (double)blocks * 4 * iters * 4 * (32.0 * 32 * 16 * 2);
  std::printf("mfma 32x32x16 bf16, register operands: %.0f TFLOP/s (%.3f ms)\n", mfma_flop / (t_m * 1e-3) / 1e12, t_m);
  std::printf("vector fp32 FMA only:                   %.3f ms\n", t_v);
  std::printf("both in every wave, VGPR accumulators:  %.3f ms  (sum of the two alone %.3f ms)\n", t_b, t_m + t_v);
  std::printf("both in every wave, AGPR accumulators:  %.3f ms\n", t_a);
  // the same split over different waves of one SIMD (one 8-wave workgroup per CU)
  auto run8 = [&](auto kern) {
    for (int w = 0; w < 3; ++w) hipLaunchKernelGGL(kern, dim3(cus), dim3(512), 0, 0, out, iters);
    CHECK(hipEventRecord(e0));
    hipLaunchKernelGGL(kern, dim3(cus), dim3(512), 0, 0, out, iters);
    CHECK(hipEventRecord(e1));
    CHECK(hipEventSynchronize(e1));
    return (double)time_ms(e0, e1);
  };
  const double x_m = run8(cross_wave<0>), x_v = run8(cross_wave<1>), x_b = run8(cross_wave<2>);
  CHECK(hipGetLastError());
  std::printf("MFMA waves alone (one per SIMD):        %.3f ms\n", x_m);
  std::printf("FMA waves alone (one per SIMD):         %.3f ms\n", x_v);
  std::printf("both, on different waves of each SIMD:  %.3f ms  (sum of the two alone %.3f ms)\n", x_b, x_m + x_v);
  const double p0 = run8(phase_mix<0>), p1 = run8(phase_mix<32>);
  CHECK(hipGetLastError());
  std::printf("both in every wave, 2 waves per SIMD:   %.3f ms in phase, %.3f ms half an iteration apart\n", p0, p1);
  std::printf("best: hbm read %.0f GB/s, hbm copy %.0f GB/s\n", best_rd, best_cp);
  mfma_random_rates(cus, 1.0, e0, e1);
  CHECK(hipFree(out));
  return 0;
}
