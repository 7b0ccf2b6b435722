// Host-side launchers of the gfx950 kernels. Each returns 0 when the launch
// was enqueued, a negative value for a configuration it does not support.
// Shapes are validated by the caller (the C ABI layer) before any launch.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>

#include "common.h"

namespace ps {

// dtype codes: 0 = fp32, 1 = bf16
struct UploadJob;
int launch_rmsnorm(int x_dt, int g_dt, int y_dt, int rows, int d, const void* x, const void* g, float eps,
                   void* y, hipStream_t st, const UploadJob* up = nullptr);

// part/splits: when splits > 1 (bf16), the QKV rows are the sum of `splits`
// fp32 split-K partials at part (see launch_gemm_split), qkv is not read
int launch_rope_kvwrite(int dt, int rows, const void* qkv, void* q_out, void* pool_layer, const SeqInfo* si,
                        const int32_t* bt, const double* inv_freq, int n_seqs, int n_q, int n_kv, int hd,
                        hipStream_t st, const float* part = nullptr, int splits = 1);
int launch_split_residual_rmsnorm(int rows, int d, int S, const float* part, const void* res, float* h,
                                  const void* g, float eps, void* y, hipStream_t st);
int launch_kv_append(int dt, int rows, const void* k, const void* v, void* pool_layer, const SeqInfo* si,
                     const int32_t* bt, int n_seqs, int n_kv, int hd, hipStream_t st);
// Pages [0, n_pages) of one sequence, all n_layers layers, copied whole from
// src_pool (its page ids src_bt) to dst_pool (dst_bt); page_bytes per page
// and layer, each pool's layer stride in bytes.
int launch_kv_copy_pages(size_t page_bytes, int n_pages, int n_layers, const void* src_pool, size_t src_layer_bytes,
                         const int32_t* src_bt, void* dst_pool, size_t dst_layer_bytes, const int32_t* dst_bt,
                         hipStream_t st);
int launch_kv_gather(int dt, int len, const void* pool_layer, const int32_t* bt, void* k_out, void* v_out,
                     int n_kv, int hd, hipStream_t st);

int launch_decode_attn(int G, int n_items, int n_kv, int n_seqs, const void* q, const void* pool_layer,
                       const SeqInfo* si, const int32_t* bt, const DecodeItem* items, float* part_o,
                       float* part_ml, const int32_t* part_begin, const int32_t* part_count, void* o,
                       float scale_log2, hipStream_t st, int max_wg = 0);  // max_wg > 0: at most that many workgroups
int launch_attn_generic(int dt, int row0, int rows, int n_seqs, int n_q, int n_kv, int hd, const void* q,
                        const void* pool_layer, const SeqInfo* si, const int32_t* bt, void* o, float scale,
                        hipStream_t st);
int compute_units();  // of the current device (256 if the query fails)
int fa_query_tile();  // query rows per prefill work item
int launch_fa_prefill(int G, int n_items, int n_kv, const void* q, const void* pool_layer, const SeqInfo* si,
                      const int32_t* bt, const PrefillItem* items, void* o, float scale_log2, hipStream_t st);

// GEMM C = epi(A W^T); ws holds split-K partials for decode-sized M.
int launch_gemm(int dtype, int r_dt, int c_dt, int epi, int M, int N, int K, const void* A, const void* W,
                const void* R, void* C, void* ws, size_t ws_bytes, hipStream_t st);
size_t gemm_workspace_bytes(int dtype, int M, int N, int K);
int launch_gemm_split(int dtype, int r_dt, int c_dt, int epi, int M, int N, int K, const void* A, const void* W,
                      const void* R, void* C, void* ws, size_t ws_bytes, hipStream_t st, int* splits);
struct SkinnyPlan {
  int wn;  // 64-row weight blocks per workgroup (1 or 2)
  int s;   // K splits
};
SkinnyPlan gemm_skinny_plan(int M, int N, int K);
int gemm_check(int dtype, int epi, int M, int N, int K);
// K splits (1..4) for a tile-path GEMM (M > 64) whose fp32 partials a fused
// consumer sums: chosen to cut the launch's rounds over the compute units,
// weighed against the partials' traffic. 1 for the skinny path.
int gemm_tile_splits(int M, int N, int K);
// Largest partial bytes gemm_tile_splits leads to for any M <= max_rows.
size_t gemm_tile_partials_bound(int max_rows, int N, int K);
// The tile GEMM's K-split partials: fp32 part[S][M][N] (A W^T over split s's
// near-equal stage range), summed in split order by the consumer.
int launch_gemm_tile_split(int M, int N, int K, int S, const void* A, const void* W, float* part, hipStream_t st);
// part[S][M][N] summed in split order plus the residual R (fp32 or bf16),
// into C (the residual epilogue of a split GEMM).
int launch_split_residual(int r_dt, int c_dt, int M, int N, int S, const float* part, const void* R, void* C,
                          hipStream_t st);
// Split-K partial bytes a launch really uses (0 when nothing is split).
size_t gemm_partials_bytes(int dtype, int epi, int M, int N, int K);
// Size of the static split-K scratch array (PS_GEMM_STATIC_SCRATCH_BYTES).
constexpr size_t kGemmStaticScratchBytes = size_t(16) << 20;
// Device address of the current GPU's copy of that array.
hipError_t gemm_static_scratch(void** out);

// model-level kernels (bf16 rows)
// One metadata upload: n16 16-byte units from mapped host memory (src) to
// dst, then each of its `blocks` workgroups stores `tag` to done[workgroup].
constexpr int kUploadMaxBlocks = 64;
struct UploadJob {
  const void* src = nullptr;
  void* dst = nullptr;
  long n16 = 0;
  uint32_t* done = nullptr;
  uint32_t tag = 0;
  int blocks = 0;  // 0: nothing to copy
};
// Workgroup b of the job (256 threads): copies its share, then stores the
// tag. Every load of src has returned before the tag store (each loaded value
// was stored to dst before the barrier), so once all `blocks` words read the
// tag the host may overwrite src. The host learns this without an event in
// the stream, whose marker would hold the next kernel back. The copy is done
// by a kernel, not a DMA-engine copy, whose start-up latency would sit
// between the previous call's last kernel and this call's first.
__device__ inline void upload_block(const UploadJob& j, int b) {
  const uint4* src = (const uint4*)j.src;
  uint4* dst = (uint4*)j.dst;
  for (long i = (long)b * 256 + threadIdx.x; i < j.n16; i += (long)j.blocks * 256) dst[i] = src[i];
  __syncthreads();
  if (threadIdx.x == 0) __hip_atomic_store(j.done + b, j.tag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}
// Fills the job for `bytes` (a multiple of 16); false for a bad size.
bool make_upload_job(const void* host_dev_ptr, void* dst, size_t bytes, uint32_t* done, uint32_t tag, UploadJob* j);
// Enqueues the job as its own kernel.
int launch_upload(const UploadJob& j, hipStream_t st);
// True when launch_rmsnorm for these types runs the kernel that can carry an
// upload job in leading workgroups of its own grid.
bool rmsnorm_carries_upload(int x_dt, int g_dt, int y_dt, int d);
int launch_embed(int rows, int d, int vocab, const void* table, const int32_t* tokens, void* x, hipStream_t st);
int launch_gather_rows(int n, int d, const void* src, const int32_t* rows, void* dst, hipStream_t st);
int launch_argmax(int rows, int vocab, const float* logits, int32_t* next, hipStream_t st);
int launch_tile_weight(int elt_bytes, long N, long K, const void* src, void* dst, hipStream_t st);

}  // namespace ps
