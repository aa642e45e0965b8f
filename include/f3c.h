/*
 * f3c — geometry-aware cached sampling of a sparse-structure flow transformer
 * (Fast3Dcache, arXiv 2511.22533) on AMD Instinct MI355X (gfx950).
 *
 * C ABI. Plain pointers and sizes only. "dev" pointers are device (HBM)
 * addresses, "host" pointers are CPU memory. Streams are HIP streams passed as
 * opaque pointers (NULL = the default stream). Every call that enqueues device
 * work is asynchronous with respect to the host, ordered on the given stream,
 * and never synchronises the device or copies device memory back to the host
 * unless its comment says so.
 *
 * Errors: every int-returning call returns F3C_OK (0) or a negative code, and
 * sets a thread-local message readable with f3c_last_error(). All arguments are
 * validated before any device work is enqueued, so a failed call has no device
 * side effects. F3C_EHIP reports a HIP runtime failure (launch or copy).
 *
 * Memory ownership: the library never allocates device memory. The caller
 * allocates the weight buffer and the state buffer (sizes from
 * f3c_model_weights_bytes / f3c_state_bytes, 256-byte aligned) and keeps them
 * alive until the model / state is destroyed. Host-side objects (f3c_model,
 * f3c_state) are owned by the library and released by the destroy calls.
 *
 * Concurrency: a model holds only its weights (read-only once loaded); every
 * buffer a step writes belongs to its state. Several states of one model may
 * therefore step concurrently on different streams. Calls on one state must
 * be ordered, normally by issuing them on one stream.
 *
 * Graph capture: f3c_state_reset, f3c_set_cond, f3c_set_uncond,
 * f3c_state_plan_times and the step calls enqueue kernels only (no
 * allocation, memset node, host copy or synchronisation), so a caller may
 * capture them in a HIP graph. The graph replays the pointers and sizes of the
 * capture: the quotas and step times are fixed at capture time.
 *
 * Layouts: latent grids and velocities are float32 [B][N][8], token-major,
 * with token n = (z*G + y)*G + x for an G x G x G grid (the flatten order of
 * the D x H x W latent, Sec. 4.2). Condition tokens are float32 [B][Nc][dc].
 */
#ifndef F3C_H
#define F3C_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define F3C_OK 0
#define F3C_EINVAL (-1)   /* bad argument, shape or value */
#define F3C_ENOMEM (-2)   /* caller-provided buffer too small */
#define F3C_EHIP (-3)     /* HIP runtime error */
#define F3C_ESTATE (-4)   /* call out of order (weights not loaded, condition not set) */

#define F3C_F32 0         /* float32 compute (debug / small models) */
#define F3C_BF16 1        /* bfloat16 operands, float32 accumulation and residual */

#define F3C_MAX_BATCH 64
#define F3C_STATE_GUIDED 1u   /* state flag: room for guided steps (two passes per sample) */
#define F3C_MAX_TOKENS 32768
#define F3C_MAX_PLAN 1024   /* times one modulation plan may hold */

typedef void* f3c_stream; /* hipStream_t */

/* Model shape. Sec. 3.2: the sparse-structure flow transformer evolves a latent
 * grid S in R^{B x C x D x H x W} under image conditioning; the per-block
 * contents follow the supplement's FLOPs list (6*D modulation, three
 * LayerNorms, self-attention, cross-attention to D_cond-wide condition tokens,
 * ratio-4 MLP). Constraints: in_ch == 8, grid^3 <= F3C_MAX_TOKENS,
 * width = heads * head_dim with head_dim in {32, 64}, width a multiple of 128
 * and at most 2048, cond_width a multiple of 64, mlp_ratio in 1..8. */
typedef struct {
  int32_t grid;
  int32_t in_ch;
  int32_t width;
  int32_t depth;
  int32_t heads;
  int32_t mlp_ratio;
  int32_t cond_tokens;
  int32_t cond_width;
  int32_t dtype;          /* F3C_F32 or F3C_BF16 */
} f3c_model_cfg;

typedef struct f3c_model f3c_model;
typedef struct f3c_state f3c_state;

/* Thread-local message describing the last failed call on this thread. */
const char* f3c_last_error(void);
int f3c_version(void);

/* ------------------------------------------------------------------ model */

/* Validate cfg and create a host-side model object. No device work. */
int f3c_model_create(const f3c_model_cfg* cfg, f3c_model** out);
void f3c_model_destroy(f3c_model* m);

/* Canonical parameter list, in load order: name (static string) and element
 * count. Linear weights are [out][in]; names ending in "_b" are biases. */
int f3c_weight_count(const f3c_model* m, int32_t* n);
int f3c_weight_info(const f3c_model* m, int32_t i, const char** name, int64_t* numel);

/* Device bytes needed for the weights of this model. */
int f3c_model_weights_bytes(const f3c_model* m, size_t* bytes);

/* Bind a caller-allocated device buffer (>= f3c_model_weights_bytes) and upload
 * the parameters of the transformer of Sec. 3.2 (per block: the modulation,
 * attention, cross-attention and MLP weights that the supplement's FLOPs list
 * counts) from host float32 arrays given in canonical order
 * (f3c_weight_info names them). Errors: F3C_EINVAL (NULL arrays, a count that
 * differs from the model's, a buffer not 256-byte aligned), F3C_ENOMEM (buffer
 * too small), F3C_EHIP (copy). Matrices are
 * rounded to the model dtype (round-to-nearest-even for bf16); biases stay f32.
 * Synchronous: returns after the upload completed. */
int f3c_model_load_weights(f3c_model* m, void* weights_dev, size_t bytes, const float* const* host_f32,
                           int32_t n);

/* FLOPs model of the supplement (FLOPs Calculation) for one forward over n_tok
 * tokens per sample, summed over blocks (modulation, 3 LN, SA, CA, MLP). */
double f3c_forward_flops(const f3c_model_cfg* cfg, int32_t n_tok, int32_t batch);

/* ------------------------------------------------------------------ state */

/* Device bytes for a sampler state of `batch` samples: the velocity cache pair,
 * activations of a full step, the per-sample condition keys/values and the
 * selection buffers. */
int f3c_state_bytes(const f3c_model* m, int32_t batch, size_t* bytes);

/* Create a state over a caller-allocated device buffer. The caches are zeroed
 * on `stream` (Algorithm 1 initialises v_cache to 0). omega defaults to 0.7. */
int f3c_state_create(f3c_model* m, int32_t batch, void* state_dev, size_t bytes, f3c_stream stream,
                     f3c_state** out);
void f3c_state_destroy(f3c_state* s);

/* As f3c_state_bytes / f3c_state_create with flags. F3C_STATE_GUIDED sizes the
 * activations and the cross-attention keys/values for two transformer passes
 * per sample (f3c_guided_step); batch is then at most F3C_MAX_BATCH / 2.
 * Unknown flags: F3C_EINVAL. */
int f3c_state_bytes_ex(const f3c_model* m, int32_t batch, uint32_t flags, size_t* bytes);
int f3c_state_create_ex(f3c_model* m, int32_t batch, uint32_t flags, void* state_dev, size_t bytes,
                        f3c_stream stream, f3c_state** out);

/* Zero both velocity caches (start of a new trajectory). Done by a kernel, not
 * a memset, so that a whole trajectory (reset, f3c_set_cond, steps) can be
 * captured in one HIP graph and replayed. */
int f3c_state_reset(f3c_state* s, f3c_stream stream);

/* SSC weight omega of Eq. (6), in [0, 1]. */
int f3c_state_set_omega(f3c_state* s, float omega);

/* Precompute the cross-attention keys/values of every block from the condition
 * tokens cond_dev (float32 [B][Nc][dc], device): the image conditioning of the
 * flow transformer (Sec. 3.2; the "Cross Attention" term of the supplement's
 * FLOPs list projects Nc condition tokens of width dc per block). They depend
 * only on the condition and the weights, so one call serves the whole
 * trajectory. Errors: F3C_EINVAL (NULL pointer). */
int f3c_set_cond(f3c_state* s, const float* cond_dev, f3c_stream stream);

/* The unconditional input of classifier-free guidance (float32 [B][Nc][dc],
 * device; an all-zero condition is the usual choice), precomputed like
 * f3c_set_cond into the second half of the keys/values. Needs a state created
 * with F3C_STATE_GUIDED (else F3C_ESTATE). */
int f3c_set_uncond(f3c_state* s, const float* uncond_dev, f3c_stream stream);

/* Modulation plan. The timestep modulation of every block (the time embedding
 * followed by the 6*width adaLN vector of each block; the "Modulation" term of
 * the supplement's FLOPs list, counted per sample and step) depends only on t
 * and the weights. f3c_state_plan_times computes it for the n times t_host[0..n-1]
 * (normally the trajectory's time grid) in ceil(n / 8) passes over the
 * modulation weights, instead of one pass per step, into the caller's device
 * buffer plan_dev (256-byte aligned, at least f3c_plan_bytes(m, n) bytes):
 * float32 [n][L][6][width] followed by [n][2][width] of time-embedding scratch.
 * A later step of this state whose t equals one of those times exactly reads
 * the planned vector; any other t computes its own as before. The planned
 * vectors are bit-identical to the ones a step computes, so planning does not
 * change results. The buffer must stay alive, and the weights unchanged, while
 * the plan is in use; calling again replaces the plan, n == 0 clears it
 * (plan_dev may then be NULL), and f3c_state_reset keeps it. The work is
 * enqueued on stream; steps on another stream must be ordered after it.
 * Errors: F3C_EINVAL (n outside 0..F3C_MAX_PLAN, a non-finite time, NULL or
 * misaligned buffer), F3C_ENOMEM (buffer too small), F3C_ESTATE (weights not
 * loaded); the previous plan is then kept. After F3C_EHIP (a launch failed)
 * the state has no plan. */
int f3c_plan_bytes(const f3c_model* m, int32_t n, size_t* bytes);
int f3c_state_plan_times(f3c_state* s, const double* t_host, int32_t n, void* plan_dev, size_t bytes,
                         f3c_stream stream);

/* One denoising step of Algorithm 1 with every token active (Phase 1, Phase 3
 * correction steps): v = G(x_t, t, c); x <- x - (t - t_next) v; caches rotate.
 * x_dev: float32 [B][N][8], updated in place. Requires t > t_next, both finite. */
int f3c_full_step(f3c_state* s, float* x_dev, double t, double t_next, f3c_stream stream);

/* One cached denoising step of Algorithm 1. n_cache_host[b] in [0, N] is the
 * number of tokens of sample b whose velocity is reused (the quota c_t of
 * Eq. 5 / Phase 3, a count of cached tokens). The c_b tokens with the lowest
 * stability score (Eq. 6; ties -> smaller token index) are cached; the
 * transformer runs on the remaining tokens only, self-attention within each
 * sample's active set; cached rows keep their stored velocity bit for bit.
 * With every n_cache_host[b] == 0 it computes exactly what f3c_full_step does. */
int f3c_cached_step(f3c_state* s, float* x_dev, double t, double t_next, const int32_t* n_cache_host,
                    f3c_stream stream);

/* One guided step (classifier-free guidance inside the guidance interval; the
 * supplement's sampling configuration uses t in [0.5, 1]). Selection as in
 * f3c_cached_step (n_cache_host == NULL: every token active), scored from the
 * stored guided velocities. The transformer runs twice on the same compacted
 * active set (the single index set of Sec. 4.2), with the condition and with
 * the unconditional input, as one batch of 2B sequences; the fresh velocity of
 * an active token is fp32(1 + w) * v_cond - fp32(w) * v_uncond, each product
 * and the difference rounded. Cached tokens keep their stored velocity. Needs a
 * F3C_STATE_GUIDED state with f3c_set_cond and f3c_set_uncond done (else
 * F3C_ESTATE); w finite. After the call, v_act (f3c_state_views) holds the
 * conditional rows [sum n_b][8] followed by the unconditional ones. */
int f3c_guided_step(f3c_state* s, float* x_dev, double t, double t_next, const int32_t* n_cache_host, double w,
                    f3c_stream stream);

/* Device views of the state (valid until the next step call):
 * v_cache / v_prev float32 [B][N][8]; idx_active int32 [sum n_b] and pos int32
 * [B][N] (packed active row or -1) of the last step's selection, both NULL
 * when the last step selected nothing (every c_b == 0: every token active in
 * token order); v_act float32 [sum n_b][8]; mod float32 [L][6][width], the
 * modulation vectors the last step read (its planned vectors when its time was
 * planned; valid while that plan is); score float32 [B][N] (written only while
 * score recording is on). act_off_host receives the B+1 active-row offsets of
 * the last step. */
int f3c_state_views(const f3c_state* s, float** v_cache, float** v_prev, int32_t** idx_active, int32_t** pos,
                    float** v_act, float** mod, float** score, int32_t* act_off_host);
int f3c_state_record_scores(f3c_state* s, int32_t on);

/* Debug: while h_trace_dev is set (device, 16-byte aligned, bytes long), every
 * step also copies the transformer's residual stream h (float32 [rows][width],
 * rows = the step's active rows, both passes on a guided step) after the
 * embedding and after each block l into slices 0 and l + 1 of h_trace_dev
 * ([L + 1][rows][width]); a step whose slices do not fit fails with
 * F3C_ENOMEM before enqueuing anything. NULL turns it off. It serves the
 * per-block parity of the transformer (the change each block makes to h). */
int f3c_state_trace_blocks(f3c_state* s, float* h_trace_dev, size_t bytes);

/* Debug: while sub_trace_dev is set (device, 16-byte aligned, bytes long),
 * every step also writes the outputs of each block's three sublayers before
 * they enter the residual stream, float32 [L][3][rows][width] (rows as for
 * f3c_state_trace_blocks): slice 3l is the self-attention output after its
 * output projection and bias, before the gate of the adaLN modulation; slice
 * 3l + 1 the cross-attention output after its projection and bias (it has no
 * gate); slice 3l + 2 the MLP output after the second linear and its bias,
 * before its gate (the block of Sec. 3.2 with the supplement's FLOPs list:
 * h += g1 * SA, h += CA, h += g2 * MLP). Each slice comes from the step's own
 * projection kernel run a second time, ungated, into the zeroed slice, so it
 * is the value the step adds. A step whose slices do not fit fails with
 * F3C_ENOMEM before enqueuing anything. NULL turns it off. */
int f3c_state_trace_sublayers(f3c_state* s, float* sub_trace_dev, size_t bytes);

/* Debug, teacher forcing of the selection (Algorithm 1: the active set I_active
 * that SSC chooses; Sec. 4.2, the transformer runs on x[:, I_active, :]): the
 * next step call of this state takes its active sets from idx_active_dev
 * (device int32, 4-byte aligned) instead of scoring and selecting them. For
 * sample b with cached count c_b its N - c_b active tokens are rows act_off[b]
 * .. act_off[b+1] - 1 (act_off the running sum of N - c_b from 0), ascending
 * token indices in [0, N); a sample with c_b == 0 lists 0 .. N-1. The step
 * copies them into the state (the idx_active view), builds pos from them and
 * consumes the hook; a step with every c_b == 0 consumes it without reading
 * the buffer. The buffer must stay valid until that step's work on its stream
 * has run. Entries outside [0, N) are clamped into range, so no access leaves
 * the state's arrays (the step's result is then unspecified); other contract
 * violations (not ascending, duplicates) also give unspecified results.
 * NULL disarms. Errors: F3C_EINVAL (NULL state, misaligned buffer). */
int f3c_debug_force_active(f3c_state* s, const int32_t* idx_active_dev);

/* Checkpoint: what Algorithm 1 carries from one step to the next besides the
 * latent x_t is the velocity cache pair (v_cache, v_prev_cache). export copies
 * v_cache then v_prev (2*B*N*8 floats, host memory owned by the caller) to
 * host; import restores them. Both synchronise `stream`. Errors: F3C_EINVAL
 * (NULL pointers), F3C_ENOMEM (n_floats below 2*B*N*8), F3C_EHIP (copy). */
int f3c_state_export(const f3c_state* s, float* host, size_t n_floats, f3c_stream stream);
int f3c_state_import(f3c_state* s, const float* host, size_t n_floats, f3c_stream stream);

/* Per-kernel-class timing with HIP events recorded around each launch of the
 * classes selected by `mask` (bit c = class c; 0 disables) on the launch
 * stream. read synchronises the recorded events and
 * returns launches, total milliseconds and total algorithmic FLOPs (dense
 * contractions: 2*M*N*K; attention: the QK^T and PV terms of the FLOPs model)
 * and algorithmic bytes (memory-bound kernels). */
#define F3C_PROF_SELECT 0
#define F3C_PROF_EMBED 1
#define F3C_PROF_MOD 2
#define F3C_PROF_LN 3
#define F3C_PROF_GEMM_QKV 4
#define F3C_PROF_ATTN_SELF 5
#define F3C_PROF_GEMM_O 6
#define F3C_PROF_GEMM_Q 7
#define F3C_PROF_ATTN_CROSS 8
#define F3C_PROF_GEMM_CO 9
#define F3C_PROF_GEMM_FC1 10
#define F3C_PROF_GEMM_FC2 11
#define F3C_PROF_FINAL 12
#define F3C_PROF_EULER 13
#define F3C_PROF_COND 14
#define F3C_PROF_CLASSES 15
int f3c_profile_enable(f3c_state* s, uint32_t mask);
int f3c_profile_read(f3c_state* s, int32_t cls, int64_t* launches, double* ms, double* flops, double* bytes);
int f3c_profile_reset(f3c_state* s);

/* ------------------------------------------------------- operator entry points
 * The individual kernels of the step on caller buffers, for parity testing of
 * each stage. Same conventions; dtype is F3C_F32 or F3C_BF16 and names the
 * element type of the "T" buffers. */

/* SSC scoring + selection (Eqs. 2, 6, 7; Algorithm 1 SSC) for B samples of N
 * tokens: v_cache, v_prev float32 [B][N][8]; n_cache_host[b] in [0, N]. Writes
 * idx_active (int32, sum(N - c_b) rows, ascending per sample), pos int32 [B][N]
 * and, if score != NULL, score float32 [B][N] (for samples with c_b > 0).
 * workspace: device scratch, 256-byte aligned, at least
 * f3c_op_select_workspace_bytes(B, N) bytes (the per-token magnitudes and the
 * partial extremes passed from the streaming scoring pass to the per-sample
 * selection); caller-owned, contents undefined after the call. Errors:
 * F3C_EINVAL (shapes, NULL or misaligned buffers, omega outside [0, 1]),
 * F3C_ENOMEM (workspace too small). */
int f3c_op_select_workspace_bytes(int32_t batch, int32_t n_tokens, size_t* bytes);
/* The selection step alone (Algorithm 1, SSC: the n_cache_host[b] tokens of
 * lowest score are cached, ties to the lower token index, NaN after every
 * number; Sec. 4.2: the active set as ascending token indices) from
 * caller-given scores, float32 [B][N] on the device, e.g. another
 * implementation's scores: a parity hook for the selection independent of
 * the scoring arithmetic. Writes idx_active and pos as f3c_op_select does;
 * needs no workspace. Errors: F3C_EINVAL (shapes, NULL pointers,
 * n_cache_host[b] outside [0, N]). */
int f3c_op_select_scores(int32_t batch, int32_t n_tokens, const float* scores, const int32_t* n_cache_host,
                         int32_t* idx_active, int32_t* pos, f3c_stream stream);
int f3c_op_select(int32_t batch, int32_t n_tokens, const float* v_cache, const float* v_prev, float omega,
                  const int32_t* n_cache_host, int32_t* idx_active, int32_t* pos, float* score, void* workspace,
                  size_t workspace_bytes, f3c_stream stream);

/* f3c_op_select without a workspace, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid allocation): the scratch lives in a fixed array in the library's
 * device code, 4 MiB + 16 KiB on each GPU, held until the process ends. It
 * serves at most F3C_NOALLOC_MAX_TOKENS tokens in all (batch * n_tokens);
 * larger calls fail with F3C_EINVAL before enqueuing anything. Nothing in it
 * needs clearing: a call overwrites what it reads. All calls on one GPU share
 * the array, so calls that overlap in time on one GPU (different streams, or
 * threads) race and must be ordered by the caller. Same arguments, results
 * and errors as f3c_op_select otherwise; the results are bit-identical to
 * it. No allocation, free or allocating library routine is called (the
 * array's address is looked up once per device with hipGetSymbolAddress). */
#define F3C_NOALLOC_MAX_TOKENS 524288
int f3c_op_select_noalloc(int32_t batch, int32_t n_tokens, const float* v_cache, const float* v_prev, float omega,
                          const int32_t* n_cache_host, int32_t* idx_active, int32_t* pos, float* score,
                          f3c_stream stream);

/* out/resid = A W^T + bias (+ epilogue). A: T [M][lda], W: T [N][ldw], bias f32 [N].
 * epilogue 0: out T [M][ldo] = value; 1: out = GELU_tanh(value);
 * 2: resid f32 [M][ldr] += (gate ? gate[n] : 1) * value.
 * Requires N % 128 == 0, K a multiple of 64 (bf16) / 32 (f32), 16-byte aligned
 * rows, ldo and ldr multiples of 4. Every output is one workgroup's sum in a
 * fixed order, so results do not depend on scheduling. */
int f3c_op_gemm(int32_t dtype, int32_t epilogue, int32_t M, int32_t N, int32_t K, const void* A, int32_t lda,
                const void* W, int32_t ldw, const float* bias, const float* gate, void* out, int32_t ldo,
                float* resid, int32_t ldr, f3c_stream stream);

/* Varlen multi-head attention: sample b's queries are rows q_off[b]..q_off[b+1]
 * of q (T, row stride ldq), its keys/values rows k_off[b]..k_off[b+1] of k/v;
 * head h uses columns h*head_dim..; o (T) gets one row per query.
 * head_dim in {32, 64}; offsets are host arrays of B+1 non-decreasing ints.
 * q_prescaled = 1 declares that q holds the queries already multiplied by
 * log2(e) / sqrt(head_dim), the softmax scale in base-2 units (as the step's
 * projections store them, rounded once); 0 for plain queries. The result is
 * softmax(Q K^T / sqrt(head_dim)) V either way (Sec. 4.2: attention over the
 * active tokens).
 * workspace (device, 16-byte aligned, may be NULL) lets launches with few
 * query tiles and long key ranges split the key range over workgroups (when
 * that shortens each wave's chain of key tiles by enough to repay the merge):
 * each split's unnormalised output, max and sum go to the workspace (splits *
 * rows * heads * (head_dim + 2) floats) and are merged in split order, so
 * results do not depend on scheduling. The split count shrinks to what the
 * workspace holds; without a workspace nothing is split. Errors: F3C_EINVAL
 * for a bad dtype, head_dim, q_prescaled, heads or batch, NULL pointers,
 * leading dims below heads*head_dim or rows not 16-byte aligned, decreasing
 * offsets, a sample with queries but no keys, a misaligned workspace, or (bf16,
 * head_dim 64) one sample's key rows, rounded up to 64, spanning 2 GiB or more. */
int f3c_op_attention(int32_t dtype, int32_t heads, int32_t head_dim, int32_t batch, const int32_t* q_off_host,
                     const int32_t* k_off_host, const void* q, int32_t ldq, const void* k, int32_t ldk,
                     const void* v, int32_t ldv, void* o, int32_t ldo, float* workspace, size_t workspace_bytes,
                     int32_t q_prescaled, f3c_stream stream);

/* out T [rows][d] = LN(h) * (1 + scale) + shift (no affine LN, eps 1e-6);
 * shift/scale f32 [d] or both NULL. d in {128, 256, 512, 1024, 2048}. */
int f3c_op_ln_mod(int32_t dtype, int32_t rows, int32_t d, const float* h, const float* shift, const float* scale,
                  void* out, f3c_stream stream);

/* Time embedding + all block modulations for time t into mod (f32 [L][6][width]). */
int f3c_op_modulation(const f3c_model* m, double t, float* mod_dev, float* scratch_dev /* 2*width f32 */,
                      f3c_stream stream);

/* Gather + embedding (Sec. 4.2: the transformer input is x at the active
 * indices; Algorithm 1 FlowTransformer input). For sample b and its r-th
 * active token i = idx_active[act_off[b] + r]:
 *   h[act_off[b] + r][:] = x[b][i][:] W_in^T + b_in + P[i][:]
 * with the model's input projection W_in, b_in and position table P.
 * x f32 [B][N][8] (N = grid^3); idx_active int32 [act_off[B]] (NULL: every
 * token active, identity order; then each segment must hold N rows);
 * act_off_host: B+1 non-decreasing host ints from act_off[0] = 0, each
 * segment 0..N rows; h f32 [act_off[B]][width]. Requires loaded weights
 * (F3C_ESTATE otherwise). */
int f3c_op_embed(const f3c_model* m, int32_t batch, const float* x, const int32_t* idx_active,
                 const int32_t* act_off_host, float* h, f3c_stream stream);

/* Final LayerNorm (no affine, eps 1e-6) and output projection (Algorithm 1
 * FlowTransformer output): v_act f32 [rows][8] = LN(h) W_out^T + b_out,
 * h f32 [rows][width]. Requires loaded weights. */
int f3c_op_final(const f3c_model* m, int32_t rows, const float* h, float* v_act, f3c_stream stream);

/* Merge, Euler update and cache rotation (Algorithm 1, update after the
 * forward): for sample b and token i, v = pos[b][i] >= 0 ? v_act[pos[b][i]] :
 * v_cache[b][i]; x[b][i] = x[b][i] - dt * v (product and difference each
 * rounded to float32, no FMA) with dt = float32(t - t_next) computed in
 * double; v_new[b][i] = v. x, v_cache, v_new f32 [B][n_tokens][8]; v_act f32
 * [act_off[B]][8] (may be NULL when no token is active); pos int32
 * [B][n_tokens] with packed rows act_off[b] + r or -1 (NULL: every token
 * active at row act_off[b] + i). v_new must not alias v_cache (the step writes
 * it over the dead v_prev). x is updated in place. */
int f3c_op_euler(int32_t batch, int32_t n_tokens, float* x, const float* v_cache, const float* v_act,
                 const int32_t* pos, const int32_t* act_off_host, double t, double t_next, float* v_new,
                 f3c_stream stream);

/* Occupancy of decoded grids (Sec. 3, voxels evolution): voxel n of grid b is
 * occupied when logits[b][n] > 0 (NaN: unoccupied). bits receives the packed
 * grid, 32 voxels per word: voxel n in bit n % 32 of word n / 32 (voxels in
 * row-major order of the grid, tail bits zero). logits f32 [B][n_voxels],
 * bits u32 [B][ceil(n_voxels / 32)], both device. batch 1..65535. */
int f3c_op_pack_occupancy(int32_t batch, int64_t n_voxels, const float* logits, uint32_t* bits,
                          f3c_stream stream);

/* Dynamic voxels, Eq. (1): counts[b] = sum over voxels of O_next XOR O_prev,
 * i.e. popcount of the XOR of the packed grids b of occ_next and occ_prev
 * (u32 [B][n_words], device; tail bits must match, e.g. both zero as written
 * by f3c_op_pack_occupancy). counts: int64 [B], device. The count of the
 * grids decoded at the anchor step and the step before it is the sigma of
 * the predictive schedule (f3c_schedule_plan). */
int f3c_op_dynamic_voxels(int32_t batch, int64_t n_words, const uint32_t* occ_next, const uint32_t* occ_prev,
                          int64_t* counts, f3c_stream stream);

/* ----------------------------------------------------------- host schedules */

/* Timestep grid t_k = shift(1 - (k-1)/T), k = 1..T+1 (Eq. S1 with factor eta;
 * eta = 1 is uniform). out_host receives T+1 doubles. */
int f3c_time_grid(int32_t steps, double eta, double* out_host);

/* ceil(steps * rho) for a decimal ratio rho (Algorithm 1: the anchor step
 * ceil(T rho_a) ending Phase 1 and the step ceil(T rho_CFG-OFF) starting
 * Phase 3). The paper gives the ratios as decimals, so rho stands for the
 * shortest decimal that rounds to the double (0.2 is 1/5 exactly,
 * 0.2000000001 is 2000000001 / 10^10) and the ceiling is exact on it, in
 * integer arithmetic: f3c_ceil_ratio(25, 0.2) = 5, f3c_ceil_ratio(25,
 * 0.2000000001) = 6. steps <= 0, rho <= 0 or NaN give 0; results above
 * INT32_MAX saturate. */
int32_t f3c_ceil_ratio(int32_t steps, double rho);

/* Whether a step starting at time t is guided: 1 when lo <= t <= hi (the
 * guidance interval of the supplement's sampling configuration, [0.5, 1] by
 * default in TRELLIS; [0, 1] is continuous guidance), else 0. */
int32_t f3c_guidance_active(double t, double lo, double hi);

/* Eqs. (4)-(5): floor(N - sigma * exp(mu * (k - k_anchor)) / gamma_up) clamped to [0, N]. */
int32_t f3c_pcsc_quota(int32_t k, int32_t n_tokens, double sigma, double mu, int32_t k_anchor, double gamma_up);

/* Algorithm 1, step 1: cached count for step k (1-based): 0 in Phase 1
 * (k <= ceil(T rho_a)); n_cache_phase2 in Phase 2 (k < ceil(T rho_off));
 * in Phase 3, 0 when (k - ceil(T rho_off) + 1) mod f_corr == 0 (f_corr > 0),
 * else floor(N * xi). The ratios are read as decimals and the ceilings and
 * the floor are exact, as in f3c_ceil_ratio. */
int32_t f3c_phase_quota(int32_t k, int32_t steps, int32_t n_tokens, int32_t n_cache_phase2, double rho_a,
                        double rho_off, double xi, int32_t f_corr);

/* Error Accumulation Elimination (Algorithm 1, SSC: the cached set is emptied
 * once "consecutive caches >= tau"). consecutive counts the immediately
 * preceding steps that ran with a non-empty cached set. Two readings:
 * F3C_TAU_CYCLE, the prose's full refresh every tau steps (tau - 1 cached
 * steps, then a full one; tau = 1 never caches), and F3C_TAU_LITERAL, the
 * algorithm's threshold (tau cached steps, then a full one; tau = 1
 * alternates). tau = 0 disables it. Returns 1 when the step must run full. */
#define F3C_TAU_CYCLE 0
#define F3C_TAU_LITERAL 1
int32_t f3c_tau_forces_full(int32_t consecutive, int32_t tau, int32_t reading);

/* Hyperparameters of the three-phase schedule (Sec. 4; defaults of the paper:
 * rho_a 0.2, rho_off 0.75, xi 0.7, f_corr 3, mu -0.07, tau 3). */
typedef struct {
  int32_t steps;        /* T */
  int32_t n_tokens;     /* N = D^3 */
  double rho_a;         /* Phase 1 ends at step ceil(T rho_a) (the anchor) */
  double rho_off;       /* Phase 3 starts at step ceil(T rho_CFG-OFF) */
  double xi;            /* Phase 3 cached ratio */
  int32_t f_corr;       /* Phase 3 correction period (0: none) */
  double mu;            /* slope of the predictive curve (Eq. 4) */
  double gamma_up;      /* latent-to-decoded volume factor of Eq. (5), > 0 */
  int32_t tau;          /* Error Accumulation Elimination interval (0: off) */
  int32_t tau_reading;  /* F3C_TAU_CYCLE or F3C_TAU_LITERAL */
} f3c_schedule_cfg;

/* The whole schedule, pre-calculated before the loop (Algorithm 1): for
 * k = 1..T, n_cache_out[k-1] = the cached count of step k from the phase rule
 * with the Phase 2 budget of Eqs. (4)-(5) (sigma: dynamic voxels measured at
 * the anchor step), then the tau constraint over the run of cached steps.
 * n_cache_out: host array of T ints. Returns F3C_EINVAL on bad parameters. */
int f3c_schedule_plan(const f3c_schedule_cfg* cfg, double sigma, int32_t* n_cache_out);

#ifdef __cplusplus
}
#endif

#endif /* F3C_H */
