/*
 * ps.h — C ABI of the MI355X (gfx950) prefill / decode hot path of a dense
 * GQA decoder layer over a paged KV cache.
 *
 * What the calls compute. The paper's serving phases (§II-B "LLM Serving
 * Phases and Their Metrics") are prefill — attention over every prompt token
 * at once, compute-bound — and decode — one token per sequence per step,
 * bound by reading the KV cache — with reasoning adding a long "think"
 * decode before the visible answer. §III-B's roofline argument and App. B.2
 * (eqs. flops-layer, bytes-layer) count the work of one layer of such a
 * model. The layer is the Llama-family pre-norm layer of the models served
 * in the evaluation:
 *
 *   xn = RMSNorm(x) * g_attn;  q,k,v = xn W_qkv^T;  q,k = RoPE(q,k, pos)
 *   o  = causal GQA softmax attention of q over the sequence's keys 0..pos
 *   h  = x + o W_o^T;  hn = RMSNorm(h) * g_ffn
 *   out = h + (silu(hn W_g^T) * (hn W_u^T)) W_d^T
 *
 * RoPE is rotate-half (pairs j, j+hd/2; angle pos * theta^(-2j/hd)); query
 * head h reads KV head h / (n_q/n_kv); attention scale 1/sqrt(hd); RMSNorm
 * puts eps inside the square root.
 *
 * The per-stage KV reservation of §IV-A (each request's KV "chunk size" in
 * tokens, CS_i) is ps_kv_alloc; the prefill / think / answer request model
 * (§IV-A PTA disaggregation) is the ps_phase tag of ps_decode_step.
 *
 * Conventions for every entry point:
 *  - Device buffers are caller-owned (e.g. torch tensors). The library never
 *    allocates device memory; it owns only host-side metadata and a small
 *    pinned host staging ring used to upload per-call metadata. Weight
 *    pointers are borrowed for the duration of the call.
 *  - Work is enqueued asynchronously on the caller's stream (a hipStream_t
 *    passed as void*; NULL = the null stream). Nothing synchronises
 *    implicitly, except that reuse of a staging slot waits on the host for
 *    the upload that last used it (a small kernel reading the pinned slot,
 *    which then stores a done tag into pinned host memory; the wait fails
 *    with PS_E_HIP after 60 s). Destroying a KV handle waits up to 10 s for
 *    its outstanding uploads, and leaves the ring allocated if they have not
 *    run by then.
 *  - Device buffers (activations, weights, KV pool, workspace) must be
 *    16-byte aligned: kernels move them with 16-byte vector accesses.
 *    Unaligned pointers are rejected with PS_E_INVALID.
 *  - Every function returns ps_status. Arguments, shapes and KV capacity are
 *    validated on the host before anything is enqueued; on any error no work
 *    is enqueued and KV metadata is unchanged. ps_last_error() returns a
 *    thread-local message for the last failing call on this thread.
 *  - A handle is not thread-safe; distinct handles are independent.
 *  - Activations and the embedding table are row-major. Linear weights use
 *    the W[out, in] convention (y = x W^T) and are stored TILED: 64 x 64
 *    tiles, tile (i, j) = W[64i .. 64i+63, 64j .. 64j+63] at tile index
 *    i * ceil(in/64) + j, each tile row-major; rows/columns past the edge of
 *    W are zero. Element W[n, k] is at
 *      ((n / 64) * ceil(in / 64) + k / 64) * 4096 + (n % 64) * 64 + k % 64.
 *    ps_tile_weight (host) and ps_op_tile_weight (device) convert a
 *    row-major matrix. Tiles make every 64-row x 64-column slab a GEMM
 *    streams one contiguous block of HBM.
 *  - bf16 buffers hold IEEE bfloat16 bit patterns.
 */
#ifndef PS_H
#define PS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t ps_status;
#define PS_OK 0
#define PS_E_INVALID 1     /* bad argument, shape, handle, sequence or layer    */
#define PS_E_NO_PAGES 2    /* KV pool has too few free pages for a reservation   */
#define PS_E_CAPACITY 3    /* write beyond a sequence's reserved capacity, or a
                              sequence would exceed max_pages_per_seq            */
#define PS_E_HIP 4         /* a HIP runtime call or launch failed                 */
#define PS_E_UNSUPPORTED 5 /* valid request the library does not implement        */

#define PS_PAGE_TOKENS 16  /* tokens per KV page                                  */
#define PS_GATE_UP_BLOCK 32 /* row-interleave granularity of w_gate_up            */

typedef enum { PS_F32 = 0, PS_BF16 = 1 } ps_dtype;

/* Request phase (§IV-A): prefill, reasoning "think" decode, answer decode.
 * The phase may change scheduling (split-K granularity) but never the
 * definition of the result. */
typedef enum { PS_PHASE_PREFILL = 0, PS_PHASE_THINK = 1, PS_PHASE_ANSWER = 2 } ps_phase;

typedef struct {
  int32_t hidden;      /* d                                  */
  int32_t n_q_heads;   /* n_q                                */
  int32_t n_kv_heads;  /* n_kv, divides n_q                  */
  int32_t head_dim;    /* hd: 64 or 128                      */
  int32_t ffn;         /* F, SwiGLU width                    */
  float rms_eps;
  double rope_theta;
  int32_t dtype;       /* ps_dtype of weights, activations and KV */
} ps_layer_cfg;

/* One layer's device weights, all in cfg.dtype; the four matrices are
 * tiled (see the conventions above):
 *   attn_norm, ffn_norm  [d]
 *   w_qkv      [d_q + 2 d_kv, d]  rows: Wq (head-major), then Wk, then Wv
 *   w_o        [d, d_q]
 *   w_gate_up  [2F, d]  Wg and Wu rows interleaved in blocks of
 *              PS_GATE_UP_BLOCK (= 32) rows: block 2i = Wg rows
 *              [32i, 32i+32), block 2i+1 = Wu rows [32i, 32i+32)
 *              (see ps_pack_gate_up), then tiled
 *   w_down     [d, F]                                                    */
typedef struct {
  const void *attn_norm, *w_qkv, *w_o, *ffn_norm, *w_gate_up, *w_down;
} ps_layer_w;

typedef struct ps_kv ps_kv;
typedef struct ps_layer ps_layer;

const char* ps_last_error(void);
const char* ps_version(void);

/* What the HIP runtime reports for one device (hipGetDeviceProperties), for
 * deriving roofline peaks on the machine at hand: the paper's roofline
 * argument (§III-B) prices work against the device's own compute and memory
 * peaks. Host-only; PS_E_HIP when the runtime has no such device. */
typedef struct {
  int32_t compute_units;      /* multiProcessorCount                        */
  int32_t clock_khz;          /* peak engine clock                          */
  int32_t memory_clock_khz;   /* peak memory clock                          */
  int32_t memory_bus_bits;    /* memory bus width                           */
  int64_t total_memory;       /* bytes                                      */
  int32_t l2_bytes;
  int32_t lds_bytes_per_block;
  char arch[64];              /* gcnArchName, NUL-terminated                */
} ps_device_info;
ps_status ps_get_device_info(int32_t device, ps_device_info* out);

/* Host helper: interleave Wg [F, d] and Wu [F, d] (host memory, elt_bytes
 * per element) into the w_gate_up row order above; out has 2F*d elements.
 * Pure layout, no arithmetic. F must be a multiple of PS_GATE_UP_BLOCK. */
ps_status ps_pack_gate_up(const void* wg, const void* wu, int32_t F, int32_t d, int32_t elt_bytes,
                          void* out);

/* Elements of the tiled form of an N x K weight: ceil(N/64) ceil(K/64) 4096
 * (0 for non-positive sizes). */
size_t ps_tiled_weight_elems(int32_t N, int32_t K);

/* Host helper: row-major w [N, K] (host memory, elt_bytes = 2 or 4 per
 * element) -> tiled `out` of ps_tiled_weight_elems(N, K) elements, padding
 * zeroed. Pure layout, no arithmetic. */
ps_status ps_tile_weight(const void* w, int32_t N, int32_t K, int32_t elt_bytes, void* out);

/* The same conversion on the device: w and out are device buffers of
 * dtype (ps_dtype), out of ps_tiled_weight_elems(N, K) elements and not
 * overlapping w. Enqueued on stream; no arithmetic. */
ps_status ps_op_tile_weight(int32_t dtype, int32_t N, int32_t K, const void* w, void* out, void* stream);

/* ------------------------------------------------------------------ KV pool
 * Device layout of the caller-provided pool (cfg.dtype elements):
 *   [n_layers][n_pages][n_kv][ K: 16 tokens x hd | V^T: hd x 16 tokens ]
 * i.e. per (layer, page, kv head) a 16 x hd block of keys, token-major, then
 * the same 16 tokens' values stored dimension-major. Token t of a sequence
 * lives in page block_table[t / 16] at slot t % 16. The block table is the
 * same for every layer. Pages are handed out from a free list whose initial
 * order is a seeded permutation (seed 0 = identity order), so logical and
 * physical order differ; results never depend on placement.
 */
size_t ps_kv_pool_bytes(const ps_layer_cfg* cfg, int32_t n_layers, int32_t n_pages);

/* Host-only: creates the metadata. `pool` is borrowed until destroy and not
 * touched by this call. A pool is the KV capacity of one instance: §III-C
 * (Observation 3) bounds decode concurrency by the bytes each token pins
 * (320 KiB per token for a 70B-class model), and §IV-A gives each stage pool
 * (prefill / think / answer) its own. */
ps_status ps_kv_create(const ps_layer_cfg* cfg, int32_t n_layers, int32_t n_pages, int32_t max_seqs,
                       int32_t max_pages_per_seq, void* pool, uint64_t page_order_seed, ps_kv** out);
ps_status ps_kv_destroy(ps_kv* kv);

/* Host-only metadata calls. ps_kv_alloc is the per-request, per-stage KV
 * reservation in tokens (the "KV chunk size" CS_i of §III-B's design-space
 * table and §IV-A: CS_T for think, CS_A for answer); PS_E_NO_PAGES when the
 * free pages cannot cover it, with nothing reserved. */
ps_status ps_kv_seq_open(ps_kv* kv, int32_t* seq);                 /* new empty sequence id        */
ps_status ps_kv_alloc(ps_kv* kv, int32_t seq, int32_t n_tokens);   /* reserve: capacity >= len + n */
ps_status ps_kv_commit(ps_kv* kv, int32_t n_seqs, const int32_t* seqs, const int32_t* n_tok);
                                                                   /* len += n (once per model step,
                                                                      after every layer wrote)    */
ps_status ps_kv_truncate(ps_kv* kv, int32_t seq, int32_t new_len); /* len = new_len <= len; keeps
                                                                      the reservation             */
ps_status ps_kv_free(ps_kv* kv, int32_t seq);                      /* return pages, close seq      */
ps_status ps_kv_seq_len(const ps_kv* kv, int32_t seq, int32_t* len);
ps_status ps_kv_capacity(const ps_kv* kv, int32_t seq, int32_t* tokens);
ps_status ps_kv_free_pages(const ps_kv* kv, int32_t* n);
ps_status ps_kv_block_table(const ps_kv* kv, int32_t seq, int32_t* pages, int32_t cap, int32_t* n);

/* Device calls. `ws` is caller-provided device workspace of ws_bytes bytes
 * (at least ps_workspace_bytes for the call's size).
 *
 * ps_kv_append (§II-B decode: every generated token's keys and values join
 * the cache that later steps read): write caller K and V rows (already
 * rotated keys) for `layer` at positions [len, len + n_tok[i]) of each
 * sequence; k, v are [sum n_tok, n_kv, hd] device arrays, rows grouped by
 * sequence in order. Does not change len (see ps_kv_commit). Errors: capacity
 * not reserved (PS_E_CAPACITY), bad layer or sequence (PS_E_INVALID).
 * ps_kv_gather (§V "What does KV transfer cost": the think -> answer handoff
 * moves a sequence's KV state out of one pool): copy positions [0, len) of
 * one sequence and layer into contiguous k_out, v_out [len, n_kv, hd]. Both
 * are bit-exact copies through the block table. */
ps_status ps_kv_append(ps_kv* kv, int32_t layer, int32_t n_seqs, const int32_t* seqs,
                       const int32_t* n_tok, const void* k, const void* v, void* ws, size_t ws_bytes,
                       void* stream);
ps_status ps_kv_gather(ps_kv* kv, int32_t layer, int32_t seq, void* k_out, void* v_out, void* ws,
                       size_t ws_bytes, void* stream);

/* Think -> answer handoff between two pools (§IV-A: a reasoning request's
 * think and answer stages run on their own pools; §V "What does KV transfer
 * cost": each such request moves its KV state once, think to answer). Copies
 * positions [0, len) of src_seq, every layer, from pool `src` into dst_seq of
 * pool `dst` and makes len the destination's committed length. Both pools
 * live on the current GPU and have the same configuration and layer count;
 * dst_seq must be open, empty and have capacity >= len reserved (ps_kv_alloc:
 * the answer stage's reservation), else PS_E_INVALID / PS_E_CAPACITY with
 * nothing changed. Pages are copied whole through both block tables, so the
 * copy is bit-exact whatever either pool's page placement; `ws` holds the two
 * page lists (8 bytes per page). The source keeps its pages: free them once
 * any later writer of those pages is ordered after the copy. src may equal
 * dst (a copy into another sequence of the same pool). */
ps_status ps_kv_transfer(ps_kv* src, int32_t src_seq, ps_kv* dst, int32_t dst_seq, void* ws, size_t ws_bytes,
                         void* stream);

/* ------------------------------------------------------------- admission
 * Per-stage KV reservation and admission for one stage pool (a ps_kv). Each
 * stage reserves its own KV "chunk size" per request in tokens (§IV-A: CS_T
 * for think, CS_A for answer; §III-B's design-space table: 512 / 1024 /
 * 2048), and PSRoute sets it from the lengths the stage actually produced,
 * admitting by observation instead of predicting lengths (§IV-D "PSRoute:
 * adaptive admission instead of prediction"):
 *   CS_i = mean of the last `window` completed requests' stage lengths,
 *          rounded up to a page and clamped to [cs_min, cs_max]
 *          (cs_initial before the first completion);
 *   admit: a request with ctx tokens of context is admitted iff a sequence
 *          slot is free and the free pages cover ctx + CS_i tokens, which
 *          are reserved (ps_kv_alloc) for a new sequence;
 *   grow:  a running sequence that outgrows its reservation takes further
 *          whole chunks of the current CS_i; when the pool cannot cover them
 *          the most recently admitted sequence is preempted (pages freed,
 *          its request goes back to the caller's queue) -- the KV thrashing
 *          the adaptive chunk size keeps rare;
 *   finish: the request's stage length joins the window; its pages are freed.
 * The scheduler decides and reserves (host only); the caller runs the steps
 * and commits lengths with ps_kv_commit. It manages only the sequences it
 * admitted. cs_initial, cs_min and cs_max are positive multiples of 16,
 * cs_min <= cs_max, window >= 1. Not thread-safe. */
typedef struct ps_sched ps_sched;
typedef struct {
  int32_t window;
  int32_t cs_initial;
  int32_t cs_min;
  int32_t cs_max;
} ps_sched_cfg;
ps_status ps_sched_create(ps_kv* kv, const ps_sched_cfg* cfg, ps_sched** out);
ps_status ps_sched_destroy(ps_sched* s);
ps_status ps_sched_chunk_size(const ps_sched* s, int32_t* cs);
ps_status ps_sched_running(const ps_sched* s, int32_t* n);
/* *seq = the admitted sequence, or -1 (not admitted, nothing changed);
 * PS_E_CAPACITY when ctx + CS_i exceeds max_pages_per_seq pages. */
ps_status ps_sched_admit(ps_sched* s, int32_t ctx_tokens, int32_t* seq);
/* Before a step adding n_tok[i] tokens to seqs[i]: extends reservations,
 * preempting as needed; writes the preempted (freed) sequence ids, in
 * preemption order, to `preempted` (room for cap >= the pool's max_seqs ids)
 * and their number to *n_preempted. Never fails for lack of pages; validates
 * every argument before changing anything. */
ps_status ps_sched_reserve_step(ps_sched* s, int32_t n, const int32_t* seqs, const int32_t* n_tok,
                                int32_t* preempted, int32_t cap, int32_t* n_preempted);
ps_status ps_sched_finish(ps_sched* s, int32_t seq, int32_t stage_tokens);

/* ------------------------------------------------------ frequency control
 * Vote-commit DVFS daemon, one per GPU (§V "How is GPU frequency actually
 * set", Alg. 1): a request entering a stage votes (target frequency f*,
 * SLO-class weight w); leaving retracts the vote. Each tick picks, over the
 * DVFS ladder, the frequency maximising sum_votes w * b(f; f*) with
 *   b(f; f*) = -(under_weight * max(0, f* - f) + over_weight * max(0, f - f*))
 * (running below a target risks the SLO, above it wastes power; ties take the
 * lower frequency; no votes give the lowest), calls `lock` only when the
 * choice changed, and calls `limit` with the power cap every tick (the
 * hardware backstop). The actuators are caller callbacks (a clock lock and a
 * power limit through the platform's management library, or test fakes);
 * they must not call back into the daemon, and return 0 on success.
 * ps_dvfs_start runs ticks on a background thread every period_ms (the
 * paper's 50-100 ms); ps_dvfs_stop joins it. Votes may come from any thread.
 * ladder_mhz is strictly increasing. Returns PS_E_HIP if an actuator failed. */
typedef int32_t (*ps_dvfs_lock_fn)(void* ctx, int32_t mhz);
typedef int32_t (*ps_dvfs_limit_fn)(void* ctx, int32_t watts);
typedef struct ps_dvfs ps_dvfs;
ps_status ps_dvfs_create(const int32_t* ladder_mhz, int32_t n, double under_weight, double over_weight,
                         int32_t power_limit_w, int32_t initial_mhz, ps_dvfs_lock_fn lock, ps_dvfs_limit_fn limit,
                         void* ctx, ps_dvfs** out);
ps_status ps_dvfs_destroy(ps_dvfs* d);
ps_status ps_dvfs_vote(ps_dvfs* d, int64_t request, int32_t target_mhz, double weight);
ps_status ps_dvfs_retract(ps_dvfs* d, int64_t request);
ps_status ps_dvfs_tick(ps_dvfs* d, int32_t* mhz, int32_t* changed);
ps_status ps_dvfs_start(ps_dvfs* d, int32_t period_ms);
ps_status ps_dvfs_stop(ps_dvfs* d);

/* PSOpt per demand-response epoch (§IV-C "Joint formulation", eq. dual;
 * App. B.1 eqs. lagrangian, kkt-f, dcap-df; §IV-C eq. rank). For each
 * stage-class group i with k GPUs at frequency f (MHz):
 *   capacity C(f) = c k^nu (1 - gamma + gamma f / f_max)  (eq. dcap-df slope)
 *   power    k (c2 f^3 + c1 f + c0)                         (§IV-C)
 *   impact   I(C) = (1/lam) int_C^C0 p(l) (l - C) dl, l ~ Normal(lam, sigma),
 *            C0 = C(f_max)                                  (§IV-B)
 * minimise sum_i w_i I_i + dt sum_i k_i P_i subject to sum_i k_i P_i <= p_max
 * and I_i <= delta_i, f_min <= f_i <= f_max, GPU counts given. The relaxation
 * is convex; the solver meets its KKT conditions directly: per group the
 * frequency stationarity of eq. kkt-f by bisection (raised to the lowest
 * frequency meeting the impact bound, whose multiplier eta follows), the
 * power-cap multiplier mu by bisection. out[i]: the relaxed optimum f, eta,
 * the impact, the ranking key of eq. rank (impact per watt reclaimed), and
 * f_step: the projection onto the ladder (rounded up, then lowered one step
 * at a time in ascending rank, the degradation ordering, while the cap is
 * exceeded and the bound allows). PS_E_CAPACITY when no admissible
 * frequencies meet the cap (out then holds the minimum-power point: the
 * caller consolidates GPUs or sheds load). Host only, microseconds. */
typedef struct {
  double w, delta;   /* class weight, impact bound                      */
  double k, nu;      /* GPUs, multi-GPU scaling exponent                */
  double c, gamma;   /* per-GPU capacity at f_max (req/s), compute-bound fraction */
  double lam, sigma; /* arrival rate: mean and standard deviation       */
  double c2, c1, c0; /* per-GPU power model, watts with f in MHz        */
} ps_psopt_group;
typedef struct {
  double f, eta, impact, rank;
  int32_t f_step;
} ps_psopt_result;
ps_status ps_psopt_solve(const ps_psopt_group* groups, int32_t n, double p_max, double f_min, double f_max,
                         double dt, const int32_t* ladder_mhz, int32_t n_ladder, ps_psopt_result* out, double* mu,
                         double* power_relaxed, double* power_projected);

/* ------------------------------------------------------------------ layer */
ps_status ps_layer_create(const ps_layer_cfg* cfg, ps_layer** out);
ps_status ps_layer_destroy(ps_layer* layer);

/* Upper bound on workspace bytes for any layer call with at most max_rows
 * new rows, max_seqs sequences and max_pages_per_seq pages per sequence. */
size_t ps_workspace_bytes(const ps_layer_cfg* cfg, int32_t max_rows, int32_t max_seqs,
                          int32_t max_pages_per_seq);

/* Prefill (§II-B: attention over every prompt token at once, compute-bound;
 * App. B.2 eq. flops-layer counts its work) or a chunk of one: each
 * sequence i contributes n_tok[i] rows of
 * x_in [sum n_tok, d] at positions [len_i, len_i + n_tok[i]); its K/V for
 * `layer` are written there (capacity must be reserved) and every row
 * attends causally over positions 0..pos (cached prefix included). x_out
 * [sum n_tok, d]. len is unchanged (call ps_kv_commit). */
ps_status ps_prefill(ps_layer* L, const ps_layer_w* w, ps_kv* kv, int32_t layer, int32_t n_seqs,
                     const int32_t* seqs, const int32_t* n_tok, const void* x_in, void* x_out, void* ws,
                     size_t ws_bytes, void* stream);

/* Decode (§II-B: one token per sequence per step, bound by reading the KV
 * cache; §III-C: the think phase is the same step over far longer contexts;
 * App. B.2 eqs. bytes-layer and gamma): one new row per sequence at position
 * len (its K/V appended before attention, so it attends over len + 1 keys).
 * x_in, x_out [n_seqs, d]. `phase` is PS_PHASE_THINK or PS_PHASE_ANSWER (the
 * §IV-A stage tag); it may change scheduling only, never the result. */
ps_status ps_decode_step(ps_layer* L, const ps_layer_w* w, ps_kv* kv, int32_t layer, int32_t phase,
                         int32_t n_seqs, const int32_t* seqs, const void* x_in, void* x_out, void* ws,
                         size_t ws_bytes, void* stream);

/* Mixed step (chunked prefill fused with decode; §II-B's phases served by one
 * batch, as the serving systems the paper builds on do when new requests
 * join a running decode batch). The rows are concatenated: first the chunk
 * rows of n_chunk sequences (chunk_tok[i] rows each), then one row for each
 * of n_dec decoding sequences. The norm, QKV GEMM and RoPE + KV write run
 * once over all rows; attention uses the prefill path for chunk rows and
 * the split-K decode path for decode rows. Same result as separate
 * ps_prefill and ps_decode_step calls up to rounding.
 * With more than 64 chunk rows and at most 64 decode rows (bf16, d a
 * multiple of 8 up to 8192) the call forks after the KV write: the decode
 * rows' attention and the rest of their layer (O, SwiGLU and down GEMMs)
 * go to a second stream that the layer handle creates on first use
 * (default priority, on the caller's device), joined back into `stream` by
 * an event before the call returns: the caller sees one stream's ordering.
 * A layer handle is used by one host thread at a time. */
ps_status ps_mixed_step(ps_layer* L, const ps_layer_w* w, ps_kv* kv, int32_t layer, int32_t n_chunk,
                        const int32_t* chunk_seqs, const int32_t* chunk_tok, int32_t n_dec,
                        const int32_t* dec_seqs, const void* x_in, void* x_out, void* ws,
                        size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------ model
 * A stack of n_layers layers (bf16) with token embedding, final RMSNorm,
 * LM head and greedy decoding, as served for the paper's 70B-class models
 * (§VI workloads; §III-C's 320 KiB/token is this stack's KV footprint).
 * Layer l uses layer l of the KV pool (which needs >= n_layers layers):
 *   h0 = embed[token];  h_L = layer_{L-1}(... layer_0(h0));
 *   logits = RMSNorm(h_L) * g_final · W_lmᵀ;  next = argmax (ties -> lowest id)
 * embed [vocab, d] is row-major, lm_head [vocab, d] tiled; final_norm [d];
 * `layers` is a host array
 * of n_layers weight sets (device pointers, borrowed until destroy).
 * Token ids live on the device; an id outside [0, vocab) embeds as a zero
 * row. Neither call commits: call ps_kv_commit after it.
 *
 * ps_model_prefill: every sequence's n_tok rows run through all layers
 * (cached prefix allowed, as in ps_prefill); only each sequence's last row
 * goes through the LM head: dev_next[i] is the greedy token after prompt i.
 * ps_model_decode_step: one token per sequence, as ps_decode_step.
 * dev_logits (optional, may be NULL): fp32 [n_seqs, vocab] logits. */
typedef struct ps_model ps_model;
ps_status ps_model_create(const ps_layer_cfg* cfg, int32_t n_layers, int32_t vocab, const void* embed,
                          const ps_layer_w* layers, const void* final_norm, const void* lm_head, ps_model** out);
ps_status ps_model_destroy(ps_model* model);
size_t ps_model_workspace_bytes(const ps_layer_cfg* cfg, int32_t vocab, int32_t max_rows, int32_t max_seqs,
                                int32_t max_pages_per_seq);
ps_status ps_model_prefill(ps_model* model, ps_kv* kv, int32_t n_seqs, const int32_t* seqs, const int32_t* n_tok,
                           const int32_t* dev_tokens, int32_t* dev_next, float* dev_logits, void* ws,
                           size_t ws_bytes, void* stream);
ps_status ps_model_decode_step(ps_model* model, ps_kv* kv, int32_t phase, int32_t n_seqs, const int32_t* seqs,
                               const int32_t* dev_tokens, int32_t* dev_next, float* dev_logits, void* ws,
                               size_t ws_bytes, void* stream);

/* ------------------------------------------------------------- single ops
 * Stage entry points (tests, microbenchmarks). Same ownership and error
 * rules. dtype arguments are ps_dtype; PS_F32 for fp32 buffers. */

/* y[r, :] = x[r, :] / sqrt(mean(x[r, :]^2) + eps) * g; fp32 arithmetic. */
ps_status ps_op_rmsnorm(int32_t x_dtype, int32_t g_dtype, int32_t y_dtype, int32_t rows, int32_t d,
                        const void* x, const void* g, float eps, void* y, void* stream);

/* C = epilogue(A W^T): A [M, K] row-major, W [N, K] tiled, both `dtype`
 * (bf16 uses the MFMA path, fp32 a vector path), fp32 accumulation.
 *   PS_EPI_STORE     C[M, N] (c_dtype)
 *   PS_EPI_RESIDUAL  C[M, N] = R + A W^T, R of r_dtype (R may alias C when
 *                    the dtypes match)
 *   PS_EPI_SWIGLU    W is a w_gate_up-interleaved [N, K]; C[M, N/2] =
 *                    silu(gate) * up with gate/up the de-interleaved halves
 * Decode-sized M (<= 64) splits K across workgroups and needs ws of at least
 * ps_op_gemm_workspace_bytes for its fp32 partials (0 bytes otherwise).
 * Supported: bf16 with K % 64 == 0, K < 2^21 and N % 256 == 0 (or M <= 64 and
 * N % 64 == 0); fp32 any shape; SwiGLU needs N % 64 == 0. */
#define PS_EPI_STORE 0
#define PS_EPI_RESIDUAL 1
#define PS_EPI_SWIGLU 2
size_t ps_op_gemm_workspace_bytes(int32_t dtype, int32_t M, int32_t N, int32_t K);
ps_status ps_op_gemm(int32_t dtype, int32_t r_dtype, int32_t c_dtype, int32_t epilogue, int32_t M, int32_t N,
                     int32_t K, const void* A, const void* W, const void* R, void* C, void* ws, size_t ws_bytes,
                     void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops or harnesses that forbid hipMalloc): ps_op_gemm
 * without a workspace argument. Decode-sized launches that split K keep
 * their fp32 partials in a library-owned static device array of
 * PS_GEMM_STATIC_SCRATCH_BYTES (one copy per GPU, held until the process
 * ends; its address is looked up once per device on the first call that
 * needs it). The call allocates nothing. Shapes whose partials would exceed
 * the array are rejected with PS_E_INVALID before anything is enqueued (the
 * launch plans write at most 8 MiB of partials, except SwiGLU launches with
 * N % 128 != 0, which write 4 M N bytes: N up to 65536 fits); a stream of a
 * device other than the current one is rejected. Every call on
 * one GPU shares that array: calls that overlap on one GPU (concurrent
 * streams) race; calls ordered on one stream do not. Each call overwrites
 * every partial it reads, so nothing carries over between calls. */
#define PS_GEMM_STATIC_SCRATCH_BYTES (16u << 20)
ps_status ps_op_gemm_static(int32_t dtype, int32_t r_dtype, int32_t c_dtype, int32_t epilogue, int32_t M,
                            int32_t N, int32_t K, const void* A, const void* W, const void* R, void* C,
                            void* stream);

/* RoPE + paged KV write for `layer`: qkv [rows, d_q + 2 d_kv] (cfg.dtype)
 * holds the QKV projection of rows grouped by sequence as in ps_prefill;
 * writes rotated q to q_out [rows, d_q] and rotated k and v into the pages
 * at positions [len, len + n_tok). */
ps_status ps_op_rope_kvwrite(ps_kv* kv, int32_t layer, int32_t n_seqs, const int32_t* seqs,
                             const int32_t* n_tok, const void* qkv, void* q_out, void* ws,
                             size_t ws_bytes, void* stream);

/* Causal attention of q [rows, n_q, hd] (rows grouped by sequence as in
 * ps_prefill, at positions [len, len + n_tok)) over the sequence's cached
 * keys 0..pos in the pages (the rows' own K/V must already be written).
 * o [rows, n_q * hd]. Uses the prefill kernel. */
ps_status ps_op_attention(ps_kv* kv, int32_t layer, int32_t n_seqs, const int32_t* seqs,
                          const int32_t* n_tok, const void* q, void* o, void* ws, size_t ws_bytes,
                          void* stream);

/* Split-K decode attention: one query row per sequence at position len
 * (the row's own K/V already written there, not yet committed), attending
 * over keys 0..len. q [n_seqs, n_q, hd], o [n_seqs, n_q * hd].
 * split_pages = at most that many pages per split: each sequence's pages
 * are cut into ceil(pages / split_pages) splits of near-equal size. 0 =
 * library choice: the smallest multiple of 4 pages, at least 8, that keeps
 * the workgroups (splits times KV heads) within about 1024, two
 * full rounds of the chip; one split per sequence when the batch alone
 * exceeds that. PS_E_UNSUPPORTED when the splits come to more than 65535
 * work items (one grid row each). */
ps_status ps_op_decode_attention(ps_kv* kv, int32_t layer, int32_t n_seqs, const int32_t* seqs,
                                 const void* q, void* o, int32_t split_pages, void* ws, size_t ws_bytes,
                                 void* stream);

/* The same attention as plan + run, for a step whose KV pool does not change
 * between layers (plan once, run per layer; also how a caller times the
 * attention kernels alone).
 * ps_op_decode_plan: checks the sequences, picks the splits and uploads the
 * work list (sequence records, page ids, splits) into ws on `stream`; the
 * plan is recorded on the handle, replacing any earlier one (a failed call
 * leaves none). Workspace need and errors as ps_op_decode_attention.
 * ps_op_decode_run: launches the attention of one layer from the plan
 * (q [n_seqs, n_q, hd] in the planned sequence order, o [n_seqs, n_q * hd]).
 * PS_E_INVALID without a plan, with a workspace other than the planned one,
 * or after any commit, truncate or free on the handle since the plan. The
 * planned work list must stay untouched in ws while runs use it. */
ps_status ps_op_decode_plan(ps_kv* kv, int32_t n_seqs, const int32_t* seqs, int32_t split_pages, void* ws,
                            size_t ws_bytes, void* stream);
ps_status ps_op_decode_run(ps_kv* kv, int32_t layer, const void* q, void* o, void* ws, size_t ws_bytes,
                           void* stream);

/* ps_op_decode_run with the attention launch capped at max_workgroups
 * workgroups (rounded down to a multiple of n_kv_heads, at least n_kv_heads):
 * each workgroup then walks several split items in turn, the form the mixed
 * step uses beside its prefill GEMMs. Same bits as the uncapped run (each
 * item's arithmetic does not depend on which workgroup runs it).
 * PS_E_INVALID for max_workgroups < 1; otherwise as ps_op_decode_run. */
ps_status ps_op_decode_run_capped(ps_kv* kv, int32_t layer, const void* q, void* o, void* ws, size_t ws_bytes,
                                  int32_t max_workgroups, void* stream);

/* Greedy token of each row of fp32 logits [rows, vocab] (ties -> lowest id). */
ps_status ps_op_argmax(int32_t rows, int32_t vocab, const float* logits, int32_t* next, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* PS_H */
