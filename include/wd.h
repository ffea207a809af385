/*
 * wd.h - C ABI of the MI355X windowed-denoising library (libwd.so).
 *
 * The library runs Window-Diffusion inference (arXiv 2601.20332) of a masked
 * diffusion language model on one AMD Instinct MI355X (gfx950): phases of one
 * refresh step plus normal steps, an external window that keeps the first E
 * undecoded positions (far-field positions are pruned), an internal window of
 * active positions that alone get logits, and a per-layer K/V cache that the
 * refresh step rewrites and normal steps reuse (Secs. 4.1-4.3 of the paper).
 * The standard full-sequence decoding step it accelerates (Sec. 3.1) is also
 * exported, for comparison.
 *
 * Conventions
 *  - Every function returns a wd_status (or a size); no exception crosses the
 *    ABI.  On a non-OK status wd_last_error() holds a message (per thread).
 *  - Device memory comes from the caller: packed weights (wd_model_bytes) and
 *    the per-generation workspace (wd_seq_bytes) are caller-allocated device
 *    buffers, 256-byte aligned, that the caller keeps alive until the
 *    corresponding wd_free_* call.  The library itself allocates only small
 *    host structures and pinned host staging buffers.
 *  - All work is enqueued on the HIP stream given to wd_init_model and is
 *    asynchronous, except calls documented as synchronizing.
 *  - Host arrays passed in are copied before the call returns; the caller
 *    keeps their ownership.
 *  - Positions are 0-based indices into one sequence (prompt first, then the
 *    generation region).  A batch is a set of independent sequences that
 *    step together; prompts are passed concatenated, without padding.
 */
#ifndef WD_H
#define WD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  WD_OK = 0,
  WD_ERR_INVALID_ARG = -1,   /* a NULL pointer, a size out of range, a bad shape */
  WD_ERR_OUT_OF_MEMORY = -2, /* a caller buffer is too small, or host allocation failed */
  WD_ERR_DEVICE = -3,        /* a HIP call failed */
  WD_ERR_STATE = -4,         /* the call is not valid in the object's current state */
  WD_ERR_UNSUPPORTED = -5    /* a shape or setting the kernels do not implement */
} wd_status;

enum { WD_DTYPE_F32 = 0, WD_DTYPE_BF16 = 1 };

/* Bidirectional decoder of the LLaDA / Qwen2 kind: pre-RMSNorm, Q/K/V
 * projections (optional bias), RoPE (half-rotation pairs (i, i + d/2),
 * frequency rope_theta^(-2i/d)) at absolute positions, non-causal attention
 * with grouped K/V heads (query head h reads K/V head h / (n_heads /
 * n_kv_heads)), output projection, SwiGLU FFN, final RMSNorm, untied LM head.
 * dtype WD_DTYPE_BF16: bf16 weights, fp32 accumulation, fp32 residual stream;
 * the RMSNorm outputs, Q/K after RoPE, V, the attention output and the SwiGLU
 * product are stored as bf16 (round to nearest even).  WD_DTYPE_F32: all fp32.
 * Supported: head_dim 64 or 128; n_heads a multiple of n_kv_heads; hidden,
 * n_heads*head_dim, ffn and vocab multiples of 64. */
typedef struct {
  int32_t n_layers, hidden, n_heads, n_kv_heads, head_dim, ffn, vocab;
  int32_t mask_id;   /* the [MASK] token; never chosen as a prediction */
  int32_t dtype;     /* WD_DTYPE_F32 or WD_DTYPE_BF16 */
  int32_t qkv_bias;  /* 0 or 1 */
  float rms_eps;
  float rope_theta;
  int32_t weight_fp8; /* 0 (default): weights as given.  1: the FP8-weight variant (not the
                         paper's precision; bf16 models only): wd_init_model stores every
                         projection matrix (Q/K/V, output, gate/up, down, LM head) as e4m3
                         codes with one float32 scale per output row, s = max |w| / 448, code =
                         nearest e4m3 value to w / s (ties to even); embeddings, norm gains
                         and biases stay bf16.  The GEMMs decode to bf16 and scale their fp32
                         sums. */
} wd_model_config;

/* Window settings (Sec. 4.2, Sec. 4.3): the internal window holds n_active
 * positions, the external window E = n_active + n_buffer positions; a phase
 * is refresh_every steps (one refresh step, then normal steps); each step
 * decodes unmask_per_step positions.
 *
 * stop_at_eos = 0 (the zero-initialized default) turns adaptive termination
 * off: every position is decoded and eos_id is ignored.  stop_at_eos = 1
 * turns it on (Sec. 4.2, adaptive termination) with eos_id a token id in
 * [0, vocab) other than mask_id: once a generated position e of a sequence
 * is decoded as eos_id, the sequence's live end becomes e + 1 (the first
 * such position).
 * Later positions leave the active set, the online rows and the attention
 * context at once, and phase starts take the window and prefix over
 * [0, end) only.  The sequence is finished when every position below its
 * end is decoded; later positions keep mask_id.  Sequences of a batch then
 * keep their own phase clocks, and the host reads each step's decisions
 * back (one small synchronization per step).
 *
 * buffer_refresh = 0 (default) is the paper's refresh (Sec. 4.3): a full
 * forward over [0, c) at every phase start.  buffer_refresh = 1 selects a
 * variant that is not the paper's method: the first phase refreshes [0, c);
 * each later refresh recomputes only the window W_ex and the positions
 * decoded in the previous phase, and every other row of [0, c) keeps the
 * K/V it was last given.  Not combinable with stop_at_eos. */
typedef struct {
  int32_t n_active, n_buffer, refresh_every, unmask_per_step;
  int32_t stop_at_eos, eos_id;
  int32_t buffer_refresh;
} wd_window_config;

typedef struct wd_model wd_model; /* opaque: packed weights and model shape */
typedef struct wd_seq wd_seq;     /* opaque: one batch of sequences being decoded */

/* Host-side result of one step.  positions / tokens / conf point to
 * caller-owned host arrays of batch * unmask_per_step entries; for sequence b
 * entries [b*k, b*k + n_selected) hold the decoded positions in rank order
 * (highest confidence first), the tokens written there and their confidence.
 * Unused entries are set to -1 / -1 / 0. */
typedef struct {
  int32_t step;        /* index t of the step just taken (0-based) */
  int32_t is_refresh;  /* 1 if it was the refresh step of a phase (of any sequence with
                          adaptive termination) */
  int32_t n_rows;      /* rows run through the layer stack, summed over the batch */
  int32_t n_selected;  /* positions decoded per sequence in this step (the most of any
                          sequence with adaptive termination) */
  int32_t* positions;
  int32_t* tokens;
  float* conf;
} wd_step_out;

/* ---- model ------------------------------------------------------------------ */

/* Number of weight tensors wd_init_model expects, in this order:
 *   emb [vocab, hidden];
 *   per layer: attn_norm [hidden], wq [n_heads*head_dim, hidden],
 *     wk [n_kv_heads*head_dim, hidden], wv [n_kv_heads*head_dim, hidden],
 *     (bq [n_heads*head_dim], bk [n_kv_heads*head_dim], bv [n_kv_heads*head_dim]
 *      when qkv_bias), wo [hidden, n_heads*head_dim], ffn_norm [hidden],
 *     wg [ffn, hidden], wu [ffn, hidden], wd [hidden, ffn];
 *   final_norm [hidden]; lm_head [vocab, hidden].
 * Matrices are row-major [out_features, in_features].  Returns -1 for an
 * invalid or unsupported configuration. */
int32_t wd_weight_count(const wd_model_config* cfg);

/* Shape of tensor i (rows, cols; cols = 1 for vectors).  WD_ERR_INVALID_ARG
 * for i out of range. */
wd_status wd_weight_shape(const wd_model_config* cfg, int32_t i, int64_t* rows, int64_t* cols);

/* Bytes of device memory wd_init_model needs for the packed weights; 0 for an
 * invalid or unsupported configuration. */
size_t wd_model_bytes(const wd_model_config* cfg);

/* Packs the weights into `device_buf` (caller-owned, >= wd_model_bytes) in
 * the layouts the kernels read.  `weights` holds wd_weight_count device
 * pointers, each to a tensor of the model dtype (fp32, or bf16 as uint16 bit
 * patterns) in the order above; they are only read during this call, and
 * the caller may free them once the stream has passed it.  `stream` is a
 * hipStream_t (NULL = the null stream) that every later call of this model
 * and its sequences is enqueued on.  Errors: WD_ERR_INVALID_ARG (NULL
 * pointer, n_weights mismatch), WD_ERR_UNSUPPORTED (shape), WD_ERR_OUT_OF_MEMORY
 * (buffer too small), WD_ERR_DEVICE. */
wd_status wd_init_model(const wd_model_config* cfg, const void* const* weights, int32_t n_weights,
                        void* device_buf, size_t buf_bytes, void* stream, wd_model** out);

void wd_free_model(wd_model* m); /* NULL is a no-op; sequences must be freed first */

/* ---- one generation --------------------------------------------------------- */

/* Bytes of device workspace a batch needs: token state, the K/V cache of
 * every layer for all batch positions, activations and step buffers.
 * 0 on invalid arguments. */
size_t wd_seq_bytes(const wd_model* m, const wd_window_config* win, int32_t batch,
                    const int32_t* prompt_lens, int32_t gen_len);

/* Starts a generation (Sec. 3.1 initial state): sequence b is its prompt
 * (prompt_lens[b] ids taken in order from the concatenated host array
 * prompt_ids) followed by gen_len [MASK] tokens; prompt positions count as
 * decoded and t = 0.  Uploads the state and the RoPE table; the first step
 * (wd_step or wd_full_step) starts the first phase.  `workspace` is
 * caller-owned device memory of >= wd_seq_bytes bytes; never-written K/V
 * cache rows are filled with NaN.  Synchronizes the stream.
 * Errors: WD_ERR_INVALID_ARG (ids outside [0, vocab), NULL pointers,
 * batch outside [1, 64], gen_len < 1, n_active outside [1, 64], n_buffer < 0,
 * refresh_every < 1, unmask_per_step < 1, stop_at_eos not 0 or 1, or 1
 * with eos_id not a token id other than mask_id, buffer_refresh not 0 or
 * 1), WD_ERR_UNSUPPORTED (stop_at_eos with buffer_refresh),
 * WD_ERR_OUT_OF_MEMORY (workspace too small), WD_ERR_DEVICE. */
wd_status wd_prefill_prompt(wd_model* m, const int32_t* prompt_ids, const int32_t* prompt_lens,
                            int32_t batch, int32_t gen_len, const wd_window_config* win,
                            void* workspace, size_t ws_bytes, wd_seq** out);

/* Phase start (Sec. 4.2): re-determines each sequence's external window as
 * its first E undecoded positions, the retained prefix [0, c) (c = the E-th
 * undecoded position + 1, or the sequence length when fewer remain) and
 * empties the set of positions decoded in the phase.  The next step becomes
 * the phase's refresh step.  wd_step calls it by itself when a phase is due
 * (every refresh_every steps, or when a window has no undecoded position
 * left); calling it earlier starts a phase early.  WD_ERR_STATE once every
 * position is decoded, or on a sequence driven by wd_full_step;
 * WD_ERR_UNSUPPORTED with adaptive termination (there wd_step drives each
 * sequence's phases). */
wd_status wd_slide_window(wd_seq* s);

/* Refresh (Sec. 4.3, refresh equation): a full forward over each sequence's
 * retained prefix [0, c) that rewrites the K/V cache rows of every layer and
 * keeps the active rows' final hidden states for the refresh step's logits.
 * Requires a slid phase whose refresh step has not been taken
 * (WD_ERR_STATE otherwise); WD_ERR_UNSUPPORTED with adaptive termination. */
wd_status wd_refresh_buffer(wd_seq* s);

/* One diffusion step: the update of Sec. 3.1 (predict every candidate
 * position, then decode the most confident ones), restricted to the active
 * positions of the internal window (Sec. 4.2), with the two step roles of
 * Sec. 4.3.  If a phase is due it slides and refreshes first (the refresh
 * step of Sec. 4.3: its active rows' logits come from the refresh forward).
 * On a normal step (Sec. 4.3) only the online rows (active positions and
 * positions decoded earlier in the phase) run the layer stack, overwrite
 * their own K/V rows and attend to all cached rows of [0, c).  Then logits
 * on the active positions, confidence (softmax probability of the argmax
 * token, [MASK] excluded, ties to the lowest id) and the unmask_per_step most
 * confident positions are decoded (ties to the lowest position).  `out` may be NULL (fully
 * asynchronous); otherwise the call synchronizes the stream and fills it.
 * WD_ERR_STATE when every position is already decoded.  With adaptive
 * termination each unfinished sequence takes its own kind of step (a phase
 * start with its refresh, or a normal step) within the same launches,
 * finished sequences take none, and the call always synchronizes;
 * WD_ERR_STATE once every sequence is finished. */
wd_status wd_step(wd_seq* s, wd_step_out* out);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the step
 * of wd_step, with the same kernels, launch plans and results, whose scratch
 * (split-K partials of the projections, split-KV attention partials,
 * confidence partials) lives in one static device array of the library,
 * WD_STATIC_SCRATCH_BYTES per GPU, held from the library's first use on that
 * GPU (wd_init_model resolves its address) until the process ends.  The call
 * allocates nothing and calls no allocating routine.  Before running it
 * bounds the step's scratch from its row counts and returns
 * WD_ERR_OUT_OF_MEMORY, with the sequence untouched, when the bound exceeds
 * the array (wd_step then takes the step).  Nothing in the array has to
 * start at zero; every step writes what it reads.  All calls on one GPU share
 * the array: calls that overlap in time on one GPU (other threads, other
 * streams) race.  WD_ERR_UNSUPPORTED with adaptive termination or while
 * kernel timing is enabled (it creates HIP events); otherwise the statuses
 * of wd_step. */
#define WD_STATIC_SCRATCH_BYTES ((size_t)96 << 20)
wd_status wd_step_noalloc(wd_seq* s, wd_step_out* out);

/* Standard decoding step (Sec. 3.1) for comparison: a forward over every
 * position of every sequence, logits for every undecoded position, and the
 * unmask_per_step most confident of them decoded.  With adaptive
 * termination the forward and the candidates of a sequence stop at its live
 * end.  A sequence is driven either by wd_full_step or by the windowed
 * calls, never both (WD_ERR_STATE). */
wd_status wd_full_step(wd_seq* s, wd_step_out* out);

/* Live end of each sequence (batch entries): one past the first generated
 * position decoded as eos_id, or the sequence length while there is none
 * (always the sequence length with stop_at_eos = 0).  Host state only: no
 * synchronization. */
wd_status wd_seq_ends(const wd_seq* s, int32_t* ends);

/* Synchronizes, then copies the token ids (sum of sequence lengths, sequence
 * after sequence) and the step counter to the host.  `decoded` (same length,
 * 1 = decoded) may be NULL.  Also reads the device's own checks of every step
 * taken so far (the rows and active positions it derived from the decoded
 * flags, each phase's retained prefix, and min(unmask_per_step, active)
 * undecoded positions decoded per sequence and step, all against the host's
 * schedule): WD_ERR_DEVICE, after the copies, if any of them failed.  A step
 * called with out == NULL reports nothing itself, so a caller that never asks
 * for step results learns of such a failure here. */
wd_status wd_get_state(const wd_seq* s, int32_t* tokens, uint8_t* decoded, int32_t* t);

/* on != 0: every later step also stores its active-row logits for
 * wd_debug_logits.  Off by default: with bf16 and at most 64 active rows the
 * LM head reduces each 64-entry vocabulary tile to the confidence inputs
 * (maximum, its lowest id, sum of exponentials; Section 3, the confidence
 * rule) inside the GEMM and the logits never reach memory.  The decisions
 * are the same either way.  For tests. */
wd_status wd_debug_keep_logits(wd_seq* s, int32_t on);

/* Synchronizes, then copies the last step's active-row logits (fp32,
 * [n_rows, vocab], sequence after sequence, active positions in increasing
 * order) and, when `positions` is not NULL, those rows' positions; *n_rows
 * receives the row count.  `capacity` is the number of rows the caller's
 * arrays hold (WD_ERR_OUT_OF_MEMORY if too small).  WD_ERR_STATE when the
 * last step kept no logits (none yet, or the fused LM head ran without
 * wd_debug_keep_logits).  For tests. */
wd_status wd_debug_logits(const wd_seq* s, float* logits, int32_t* positions, int32_t capacity,
                          int32_t* n_rows);

/* Synchronizes, then copies K and V of one layer and one sequence for
 * positions [0, c) as fp32 [c, n_kv_heads, head_dim] each, with c the
 * current retained prefix; *ctx_len receives c.  `capacity` is the number of
 * positions the arrays hold.  For tests. */
wd_status wd_debug_kv(const wd_seq* s, int32_t layer, int32_t b, float* k, float* v,
                      int32_t capacity, int32_t* ctx_len);

void wd_free_seq(wd_seq* s); /* NULL is a no-op; synchronizes the stream */

/* Tests only.  The values the GEMMs use for output row `row` of weight
 * tensor `tensor` (an index into the wd_init_model order; projection
 * matrices only: wq, wk, wv, wo, wg, wu, wd, lm_head), read back from the
 * packed device buffer and decoded on the host: `values` receives the row's
 * in_features weights in their original column order (bf16 values, or the
 * e4m3 values before scaling with weight_fp8) and *scale the row's fp8
 * scale (1 without weight_fp8).  Synchronizes.  WD_ERR_INVALID_ARG for an
 * index that is not a projection matrix or a row out of range;
 * WD_ERR_UNSUPPORTED for fp32 models. */
wd_status wd_debug_weight_row(const wd_model* m, int32_t tensor, int32_t row, float* values,
                              float* scale);

/* ---- kernel timing ------------------------------------------------------------- */

/* Kernel classes of the recorded GEMM launches. */
enum {
  WD_PROF_ALL = 0,        /* every recorded launch */
  WD_PROF_GEMM_ROWS = 1,  /* k_gemm_bf16 / k_gemm_bf16_fused: at most 64 rows (96 for
                             gate/up, O and down), each weight read once (normal steps,
                             LM head) */
  WD_PROF_GEMM_TILED = 2, /* more rows (refresh and full-sequence steps):
                             k_gemm_bf16_dma (bf16, widths a multiple of 256), else
                             k_gemm_bf16_big */
  WD_PROF_GEMM_F32 = 3,   /* k_gemm_f32: fp32 models */
  WD_PROF_ATTN = 4        /* bf16 attention of one layer (k_attn_bf16 and, when the keys are
                             split, k_attn_combine, timed as one unit); bytes = K and V rows
                             [0, c) of every sequence + the q rows read + the output rows
                             written, flops = 4 * rows * c * n_heads * head_dim */
};

/* When enabled, every launch of the projection GEMM kernels (Q/K/V, output,
 * gate/up, down and LM-head products) on this model's stream records a pair
 * of HIP events from its own dispatch (start and end of the kernel), and the
 * launch's kernel class and algorithmic traffic and work are recorded: bytes = weights (N*K elements) + input rows (M*K
 * elements) + what the launch writes (fp32 M*N*4 for a split-K launch, the
 * bf16 results of a fused Q/K/V or SwiGLU launch, 12 bytes per row and
 * 64-entry vocabulary tile for the fused LM head), flops = 2*M*N*K.  Up to 1 << 20 launches
 * are kept (WD_ERR_OUT_OF_MEMORY from the launching call beyond that).
 * Disabled by default; every call discards the records taken so far. */
wd_status wd_profile_enable(wd_model* m, int32_t enable);

/* Synchronizes the model's stream, then returns, over the launches of class
 * `kernel` (WD_PROF_*) recorded since profiling was last enabled, their
 * number, the sum of their event-measured durations (milliseconds) and of
 * their algorithmic bytes and flops.  Records are kept, so several classes
 * can be read.  Any output pointer may be NULL; an unknown class is
 * WD_ERR_INVALID_ARG. */
wd_status wd_profile_read(wd_model* m, int32_t kernel, int64_t* launches, double* total_ms,
                          double* alg_bytes, double* alg_flops);

/* Measures, on the model's device and stream, the achievable dense bf16
 * matrix-core throughput (a loop of independent 32x32x16 MFMAs on every CU,
 * TFLOP/s) and HBM read bandwidth (one non-temporal pass over a 4 GiB
 * buffer, GB/s); the better of two timed runs each.  Allocates and frees the
 * 4 GiB buffer itself; synchronizes.  For reporting roofline fractions
 * against measured as well as vendor peaks. */
wd_status wd_measure_peaks(wd_model* m, double* mfma_bf16_tflops, double* hbm_read_gbs);

/* ---- host-only helpers -------------------------------------------------------- */

/* The schedule's counts for one sequence, from counts alone (they do not
 * depend on which positions get decoded): for each step t, whether it is a
 * refresh step, the retained prefix length c, |A|, the rows the step runs
 * through the layer stack (c on a refresh step, |W_ex| + |D_{p-1}| on the
 * buffer-only variant's later refreshes, |A| + |D_p| otherwise) and the
 * positions it decodes.  Adaptive termination is ignored (its counts depend
 * on where <eos> is decoded).  Writes at most max_steps entries to each
 * non-NULL array and returns the total number of steps, or -1 on invalid
 * arguments.  Needs no GPU. */
int32_t wd_plan(int32_t n_prompt, int32_t gen_len, const wd_window_config* win, int32_t max_steps,
                int32_t* is_refresh, int32_t* ctx_len, int32_t* n_active, int32_t* n_rows,
                int32_t* n_decode);

/* Tests only.  The launch plan the bf16 projection GEMM takes for an
 * M x K by K x N product (fp8: fp8 weights; at most max_splits K splits),
 * as eight integers in out: the kernel (1 pipelined few-row kernel with
 * K-split partials, 2 many-row LDS-pipelined kernel, 3 split-K tiled kernel),
 * rows and features of a workgroup tile, K splits, 32-wide K steps per split,
 * workgroups, waves per workgroup, and whether the launchers accept the plan
 * (bit 0 as a plain GEMM, bit 1 with the many-row kernel's SwiGLU epilogue).
 * The step loop plans every projection this way with no split cap.
 * WD_ERR_INVALID_ARG for sizes outside [1, 2^24], K not a multiple of 32 or
 * NULL out.
 * Needs no GPU. */
wd_status wd_debug_gemm_plan(int32_t M, int32_t N, int32_t K, int32_t fp8, int32_t max_splits,
                             int32_t* out);

/* Message of the last non-OK status on this thread ("" if none). */
const char* wd_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* WD_H */
