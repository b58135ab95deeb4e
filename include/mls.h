/*
 * mls.h - fused multi-sub-model LM head + cross-entropy + distillation on
 * AMD Instinct MI355X (gfx950).
 *
 * The operation ("Matryoshka Language Model Suites", section 2, "Method"):
 * a suite of M nested sub-models, each with its own LM head W_i [V, d_i]
 * applied to its final hidden states h_i [T, d_i] (paragraphs "Modeling" and
 * "Inter-model Junction"); every sub-model takes next-token cross-entropy;
 * every sub-model except the teacher s (the largest one) adds a distillation
 * term from the teacher's stop-gradient softmax (eq. (2)); the sub-model
 * losses are combined convexly (eq. (3)) and summed.
 *
 * The library computes, for every sub-model i and valid token t
 * (label y_t != ignore_index):
 *   l_i[t]     = W_i h_i[t]                          logits, never stored
 *   CE_i       = mean_t ( logsumexp(l_i[t]) - l_i[t, y_t] )
 *   KL_i       = mean_t KL( q[t] || softmax(l_i[t] / tau) ),  KL_s = 0,
 *                q[t] = softmax(l_s[t] / tau)
 *   H          = mean_t entropy(q[t])
 * eq. (2) at temperature tau is KL_i + H. The backward pass is the exact
 * gradient of J = sum_i g_ce[i] CE_i + g_kl[i] KL_i with q held constant
 * (stop_grad): with N valid tokens,
 *   dJ/dl_i[t] = ( g_ce[i] (softmax(l_i) - onehot(y_t))
 *                + g_kl[i] / tau (softmax(l_i / tau) - q) ) / N,
 *   grad_h_i = dJ/dl_i  W_i,     grad_W_i = (dJ/dl_i)^T h_i.
 * eq. (3) with the tau^2 temperature factor is g_ce = (1 - alpha), g_kl =
 * alpha tau^2 for students and g_ce = 1, g_kl = 0 for the teacher
 * (mls_coeffs). No [T, V] tensor is ever materialised: the forward keeps
 * per-row online log-sum-exp statistics, the backward recomputes logits
 * one vocabulary chunk at a time.
 *
 * Conventions
 *  - Every device buffer is owned and allocated by the caller; the library
 *    never allocates device memory and keeps no mutable global state. Calls
 *    on different streams with different workspaces may run concurrently.
 *  - All device work is enqueued on the given stream (a hipStream_t; NULL is
 *    the default stream) and is asynchronous: buffers must stay valid until
 *    the stream reaches the enqueued work.
 *  - Argument validation is done on the host before any device call; on an
 *    error nothing is enqueued and the status says why (mls_last_error gives
 *    the detail, per thread).
 *  - Row-major layouts. Device pointers to h_i, W_i, grads and workspace must
 *    be 16-byte aligned, labels 8-byte aligned.
 */
#ifndef MLS_H_
#define MLS_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MLS_MAX_MODELS 8

typedef enum mls_status {
  MLS_OK = 0,
  MLS_INVALID_ARG = 1,          /* null pointer, bad size or index, bad tau / alpha, misalignment */
  MLS_UNSUPPORTED = 2,          /* dtype or width the kernels do not handle */
  MLS_WORKSPACE_TOO_SMALL = 3,  /* workspace_bytes below what mls_query_sizes reports */
  MLS_HIP_ERROR = 4             /* a HIP runtime call failed; mls_last_error has its text */
} mls_status;

typedef enum mls_dtype {
  MLS_BF16 = 0,  /* bfloat16 h_i and W_i, fp32 accumulation */
  MLS_F32 = 1    /* float32 h_i and W_i */
} mls_dtype;

enum mls_mode {
  MLS_MODE_PAPER = 0,    /* eq. (3): students (1-alpha) CE + alpha tau^2 KL; teacher CE */
  MLS_MODE_ADDITIVE = 1  /* students CE + alpha tau^2 KL; teacher CE */
};

enum mls_flags {
  MLS_ACCUMULATE_GRAD_W = 1u, /* grad_W_i += instead of = */
  MLS_ACCUMULATE_GRAD_H = 2u, /* grad_h_i += instead of = */
  MLS_FWD_BWD_RECOMPUTE = 4u  /* mls_distill_fwd_bwd: recompute the logits in the backward
                                 instead of storing them per token chunk */
};

/* Device-side error bits written into the statistics buffer by the forward. */
enum mls_device_flags {
  MLS_DEVFLAG_LABEL_RANGE = 1, /* a label outside [0, V) that is not ignore_index;
                                  such tokens are treated as ignored */
  MLS_DEVFLAG_NONFINITE = 2    /* some token's log-sum-exp (ignored tokens included)
                                  or a valid token's cross-entropy, KL or teacher
                                  entropy is NaN or infinite: a non-finite value in
                                  h_i or W_i. Losses of valid tokens, or the head
                                  gradients (an ignored token's h_i row still enters
                                  grad_W = G^T h), are then not meaningful. */
};

/*
 * One problem instance. Fields:
 *   M             number of sub-models, 1..MLS_MAX_MODELS
 *   teacher       index of the distillation teacher s; -1 selects M-1 (the largest)
 *   T             number of tokens (batch x sequence, flattened), >= 1
 *   V             vocabulary size, >= 2
 *   d[i]          width of sub-model i; a multiple of 8 (bf16) or 4 (f32)
 *   h[i]          device pointer, [T, d[i]] row-major, in_dtype
 *   W[i]          device pointer, [V, d[i]] row-major, in_dtype
 *   labels        device pointer, [T] int64 next-token ids
 *   ignore_index  label value that removes a token from every loss (usually -100)
 *   alpha         distillation weight of eq. (3), in [0, 1]; only used when
 *                 mls_distill_bwd is given no coefficient vectors
 *   tau           distillation temperature, finite and > 0 (1 = eq. (2) as printed)
 *   in_dtype      an mls_dtype
 *   grad_h_dtype  mls_dtype of the grad_h_i outputs of mls_distill_bwd: MLS_F32, or
 *                 MLS_BF16 (rounded once from the fp32 sums; over several
 *                 vocabulary chunks the partial sums are kept in fp32 in the
 *                 workspace). Note that 0 is MLS_BF16: a zero-filled struct asks
 *                 for bf16 gradients.
 *   flags         OR of mls_flags
 *   vocab_chunk   backward vocabulary chunk width, rounded up to a multiple of
 *                 256; 0 = chosen by the library: at least four balanced
 *                 chunks (more if one chunk's bf16 logit-gradient slabs would
 *                 pass 4 GiB), so no slab spans the whole vocabulary. On the
 *                 bf16 path (every d_i a multiple of 64) the width is also
 *                 capped so that one slab [T_pad][width] and one head chunk
 *                 [width][d_i] stay below 4 GiB (T_pad = T rounded up to 128).
 *                 A backward whose T_pad * d_i bf16 panel would reach 4 GiB
 *                 runs on the general (slower) kernels instead.
 */
typedef struct mls_problem {
  int32_t M;
  int32_t teacher;
  int64_t T;
  int64_t V;
  int64_t d[MLS_MAX_MODELS];
  const void* h[MLS_MAX_MODELS];
  const void* W[MLS_MAX_MODELS];
  const int64_t* labels;
  int64_t ignore_index;
  float alpha;
  float tau;
  int32_t in_dtype;
  int32_t grad_h_dtype;
  uint32_t flags;
  int64_t vocab_chunk;
} mls_problem;

/*
 * Sizes of the two caller-allocated device buffers for problem p.
 *   workspace_bytes  scratch for one call of mls_distill_fwd, mls_distill_bwd
 *                    or mls_diagnostics (contents are not kept between calls).
 *                    It is the largest of three needs: the forward's two
 *                    16-byte partial records per sub-model, token and 128-row
 *                    vocabulary tile; the backward's per-chunk logit-gradient
 *                    slab (normally the largest); the
 *                    diagnostics' two records of (M*M + 3M) floats per token
 *                    and 128-row vocabulary tile.
 *   stats_bytes      per-row statistics the forward writes and the backward
 *                    reads. Layout (all little-endian, offsets in elements of
 *                    float32 from the start):
 *                      lse1[M][T]   log-sum-exp of l_i[t]
 *                      lset[M][T]   log-sum-exp of l_i[t] / tau
 *                      ce_row[M][T] per-token CE (0 on ignored tokens)
 *                      kl_row[M][T] per-token KL (0 on ignored tokens and for the teacher)
 *                      h_row[T]     per-token teacher entropy (0 on ignored tokens)
 *                    followed by int32 n_valid and int32 device flags
 *                    (mls_device_flags).
 * Pure host function: no device call. Either output pointer may be NULL.
 */
mls_status mls_query_sizes(const mls_problem* p, size_t* workspace_bytes, size_t* stats_bytes);

/*
 * Forward pass. Writes the statistics buffer and the losses:
 *   ce[M], kl[M]  device float32; kl[teacher] = 0; raw values (no alpha, no tau^2)
 *   entropy       device float32 [1], mean teacher entropy H (may be NULL)
 * With no valid token every loss is 0. workspace/workspace_bytes as given by
 * mls_query_sizes. Asynchronous on stream.
 */
mls_status mls_distill_fwd(const mls_problem* p, void* stats, float* ce, float* kl,
                           float* entropy, void* workspace, size_t workspace_bytes,
                           void* stream);

/*
 * Backward pass: grad_h[i] (device [T, d[i]], float32 or bfloat16 as
 * p->grad_h_dtype says) and grad_W[i] (device float32 [V, d[i]]) of
 * J = sum_i g_ce[i] CE_i + g_kl[i] KL_i, with the teacher distribution under
 * stop_grad (paper section 2, eq. (2) and eq. (3)).
 *   stats        the buffer written by mls_distill_fwd on the same inputs
 *   g_ce, g_kl   device float32 [M] coefficient vectors (e.g. the upstream
 *                gradients of ce and kl), read on the device so no host
 *                synchronisation is needed; if both are NULL the coefficients
 *                of MLS_MODE_PAPER with p->alpha and p->tau are used. One NULL
 *                and one non-NULL is an error.
 *   grad_h       host array of M device pointers; an entry may be NULL to skip
 *                that gradient. Overwritten unless MLS_ACCUMULATE_GRAD_H (a bf16
 *                grad_h is then read, added to in fp32 and rounded once).
 *   grad_W       host array of M device pointers; an entry may be NULL.
 *                Overwritten unless MLS_ACCUMULATE_GRAD_W.
 * Asynchronous on stream.
 */
mls_status mls_distill_bwd(const mls_problem* p, const void* stats, const float* g_ce,
                           const float* g_kl, void* const* grad_h, float* const* grad_W,
                           void* workspace, size_t workspace_bytes, void* stream);

/*
 * Forward and backward in one call, for a caller that knows the objective's
 * coefficients before the forward (a training step: J = sum_i g_ce[i] CE_i +
 * g_kl[i] KL_i with eq. (3)'s coefficients, paper section 2, "Integrated
 * Distillation", eq. (2) and eq. (3)). Same outputs as mls_distill_fwd followed by
 * mls_distill_bwd with the same arguments (stats, losses, entropy, grad_h,
 * grad_W, flags and grad_h_dtype as described there; g_ce / g_kl NULL means
 * eq. (3) with p->alpha and p->tau).
 *
 * The logits are not recomputed: the tokens are taken in at least two chunks;
 * for each, the forward stores every sub-model's logits of the chunk in the
 * workspace (fp16 of each logit's distance to a local maximum over 64
 * vocabulary entries, so the entries near the maximum, which carry the
 * softmax's mass, are the most exact), the log-sum-exp rows are merged, the
 * logit gradient is formed in place (bf16) and the two head products run on it
 * (grad_h of the chunk's tokens complete, grad_W accumulated over the chunks).
 * No [T, V] array exists at any time: a chunk holds at most
 * ceil(T / 2) tokens, fewer when one sub-model's logits of a chunk would reach
 * 4 GiB or all of them 16 GiB. Problems of one 128-token tile, widths that are
 * not multiples of 64, fp32 inputs, heads [V, d_i] of 4 GiB or more, or
 * MLS_FWD_BWD_RECOMPUTE in p->flags run the forward and then the recomputing
 * backward instead. workspace_bytes: at least what mls_query_fwd_bwd_workspace
 * reports. Asynchronous on stream.
 */
mls_status mls_query_fwd_bwd_workspace(const mls_problem* p, size_t* workspace_bytes);
mls_status mls_distill_fwd_bwd(const mls_problem* p, void* stats, float* ce, float* kl,
                               float* entropy, const float* g_ce, const float* g_kl,
                               void* const* grad_h, float* const* grad_W, void* workspace,
                               size_t workspace_bytes, void* stream);

/*
 * Cross-model diagnostics (paper section 3, "Training Dynamics and Model
 * Agreement"): for every ordered pair of sub-models (i, j), over the valid
 * tokens (label != ignore_index, in range)
 *   kl_pair[i*M + j] = mean KL(softmax(l_i) || softmax(l_j))   (temperature 1)
 *   agree[i*M + j]   = mean [argmax_v l_i == argmax_v l_j]     (ties: lowest index)
 * kl_pair and agree are device float32 [M*M]; argmax (device int32 [M][T], may be
 * NULL) receives every token's top-1 index per sub-model. One pass over the
 * logits, normalised as it goes: no forward statistics are needed (tau and
 * teacher do not matter here). The workspace of mls_query_sizes suffices.
 * A pass holds at most 4 sub-models; a larger suite runs one pass per subset
 * of 4, the subsets chosen so that every pair of sub-models shares one (e.g.
 * 6 passes for M = 8), each staged in the workspace and scattered into the
 * outputs. With no valid token the outputs are 0. Asynchronous on stream.
 */
mls_status mls_diagnostics(const mls_problem* p, float* kl_pair, float* agree, int32_t* argmax,
                           void* workspace, size_t workspace_bytes, void* stream);

/*
 * Inter-model junction (paper section 2, "Inter-model Junction", eq. (1)):
 * per token t, the output o[t] (width d_prev) of sub-model m is rescaled to
 * the Euclidean norm of the fresh embedding e[t] (width d_fresh) of
 * sub-model m+1, and the two are concatenated into x[t] (width
 * d_prev + d_fresh):
 *   s = ||e[t]|| / ||o[t]||,  x[t] = [s*o[t] | e[t]]   (MLS_JUNCTION_PREV_FIRST)
 *                             x[t] = [e[t] | s*o[t]]   (MLS_JUNCTION_FRESH_FIRST)
 * PREV_FIRST puts sub-model m's channels first, as the text after eq. (1)
 * describes; FRESH_FIRST is the literal order of eq. (1). A zero norm gives
 * s = 0. Norms and dot products are accumulated in fp32.
 */
enum mls_junction_layout {
  MLS_JUNCTION_PREV_FIRST = 0,
  MLS_JUNCTION_FRESH_FIRST = 1
};
enum mls_junction_flags {
  MLS_JUNCTION_ACCUMULATE = 1u  /* backward: g_o += and g_e += instead of = */
};
typedef struct mls_junction {
  int64_t T;           /* tokens, >= 1 */
  int64_t d_prev;      /* width of o: a multiple of 8 in [8, 8192] */
  int64_t d_fresh;     /* width of e: a multiple of 8 in [8, 8192] */
  int32_t act_dtype;   /* mls_dtype of o, e and x */
  int32_t grad_dtype;  /* mls_dtype of g_x, g_o and g_e */
  int32_t layout;      /* mls_junction_layout */
  uint32_t flags;      /* mls_junction_flags */
} mls_junction;

/*
 * Forward: x = junction(o, e). o [T][d_prev], e [T][d_fresh] and x
 * [T][d_prev + d_fresh] are row-major device arrays of act_dtype, 16-byte
 * aligned; x must not overlap o or e. Asynchronous on stream.
 */
mls_status mls_junction_fwd(const mls_junction* j, const void* o, const void* e, void* x,
                            void* stream);

/*
 * Backward: with g_x [T][d_prev + d_fresh] the gradient of a loss with
 * respect to x (grad_dtype), writes
 *   g_o = s * (g - (g.o) o / ||o||^2)
 *   g_e = g_e0 + (g.o) / (||o|| ||e||) * e
 * where g and g_e0 are the blocks of g_x on the rescaled and the fresh
 * channels (ratio terms are 0 where a norm is 0). g_o [T][d_prev] and g_e
 * [T][d_fresh] are grad_dtype, 16-byte aligned, and must not overlap the
 * inputs; with MLS_JUNCTION_ACCUMULATE they are added to (the sum is formed
 * in fp32 and stored once). o and e are the forward's inputs.
 */
mls_status mls_junction_bwd(const mls_junction* j, const void* o, const void* e, const void* g_x,
                            void* g_o, void* g_e, void* stream);

/*
 * Head step of nested speculative decoding (paper section 2, paragraph
 * "Speculative Decoding"; section 3 measures greedy and nucleus top-p 0.9
 * sampling at temperature 0.4). A smaller sub-model drafts gamma tokens and a
 * larger one verifies them; each step maps hidden states to logits with that
 * sub-model's LM head and samples from them.
 *
 * Sampling distribution of a row of logits l: softmax(l / temperature), then
 * the nucleus filter keeps the most probable tokens (ties: lower index first)
 * up to and including the first one at which the kept mass reaches top_p, and
 * renormalises (top_p = 1 keeps every token). Random numbers are inputs:
 * uniforms in [0, 1). A draw with uniform u returns the smallest index whose
 * cumulative kept probability, in index order, exceeds u. Greedy mode takes
 * the argmax (lowest index on ties). Rows of up to 65536 entries.
 */
typedef struct mls_sampling {
  int64_t V;          /* vocabulary size, 2..65536 */
  float temperature;  /* > 0 (ignored when greedy) */
  float top_p;        /* in (0, 1] (ignored when greedy) */
  int32_t greedy;     /* nonzero: argmax */
  int32_t reserved;   /* 0 */
} mls_sampling;

/*
 * logits[t][v] = sum_k o[t][k] W[v][k] (fp32 row-major [T][V]) for o [T][d]
 * and W [V][d] of dtype (MLS_BF16: d a multiple of 8; MLS_F32: of 4), all
 * device arrays, 16-byte aligned. Asynchronous on stream.
 */
mls_status mls_head_logits(int64_t T, int64_t V, int64_t d, int32_t dtype, const void* o,
                           const void* W, float* logits, void* stream);

/* Bytes of one row's sampling-distribution record (an opaque device record:
 * the row's maximum, total and kept mass, nucleus threshold and tie cut). */
#define MLS_ROW_PARAMS_BYTES 20

/*
 * tokens[r] (int32, device) = a draw from row r of logits [rows][V] with
 * uniform u[r] (device [rows]; may be NULL when greedy). When params is not
 * NULL (and not greedy), row r's distribution record is also written to
 * params + r * MLS_ROW_PARAMS_BYTES (device, 4-byte aligned): a drafting loop
 * can hand these records to mls_spec_verify as draft_params.
 */
mls_status mls_sample(const mls_sampling* s, int64_t rows, const float* logits, const float* u,
                      int32_t* tokens, void* params, void* stream);

/* Workspace bytes of mls_spec_verify for a batch and draft length (enough
 * with or without draft_params). */
mls_status mls_spec_verify_workspace(int64_t batch, int64_t gamma, size_t* bytes);

/*
 * Speculative verification of `batch` sequences with `gamma` >= 0 drafted
 * tokens each (device arrays). The draft's arrays are in drafting order, one
 * [batch] slice per draft step, as a drafting loop produces them:
 *   draft_logits  [gamma][batch][V]      the draft's logits at each drafted position
 *   draft_tokens  [gamma][batch] int32   the drafted tokens
 *   u_accept      [gamma][batch]         uniforms of the acceptance tests
 *   target_logits [batch][gamma + 1][V]  the verifier's logits at the drafted positions
 *                                        and the one after them (one pass per sequence)
 *   u_sample      [batch]                uniform of the final draw
 * Per sequence, drafted token x at position k is kept when
 * u_accept * q(x) < p(x) (q: the draft's sampling distribution, p: the
 * verifier's). At the first rejection, next_token is drawn from max(0, p - q)
 * renormalised and n_accepted = k; if all are kept, n_accepted = gamma and
 * next_token is drawn from the verifier's distribution at position gamma.
 * Greedy mode keeps a token while it equals the verifier's argmax and emits
 * the verifier's argmax (u_accept, u_sample and the workspace may be NULL).
 * draft_params (device, may be NULL): [gamma][batch] records of
 * MLS_ROW_PARAMS_BYTES from mls_sample on the same draft rows with the same
 * sampling settings; then the draft rows' distributions are not recomputed.
 * Outputs n_accepted, next_token: int32 [batch]. Asynchronous on stream.
 */
mls_status mls_spec_verify(const mls_sampling* s, int64_t batch, int64_t gamma,
                           const float* draft_logits, const float* target_logits,
                           const int32_t* draft_tokens, const float* u_accept,
                           const float* u_sample, const void* draft_params,
                           int32_t* n_accepted, int32_t* next_token, void* workspace,
                           size_t workspace_bytes, void* stream);

/*
 * mls_spec_verify without a workspace, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops). Same arguments,
 * semantics and kernels as mls_spec_verify; the per-row distribution records
 * (MLS_ROW_PARAMS_BYTES each, batch * (2 gamma + 1) of them) live in a static
 * device array of MLS_SPEC_VERIFY_STATIC_BYTES that the library keeps on each
 * device it runs on until the process ends. Problems needing more than that
 * (mls_spec_verify_workspace reports the need) are rejected with
 * MLS_INVALID_ARG before any device work. The call itself allocates nothing
 * (its first call on a device looks up that device's copy of the array). All
 * calls on one device share the array: calls that may overlap on one device
 * (different streams, or different host threads, without ordering between
 * them) race and must not be issued; calls ordered on one stream are safe.
 */
#define MLS_SPEC_VERIFY_STATIC_BYTES (2u << 20)
mls_status mls_spec_verify_noalloc(const mls_sampling* s, int64_t batch, int64_t gamma,
                                   const float* draft_logits, const float* target_logits,
                                   const int32_t* draft_tokens, const float* u_accept,
                                   const float* u_sample, const void* draft_params,
                                   int32_t* n_accepted, int32_t* next_token, void* stream);

/*
 * Host helper: loss coefficients of the objective (host arrays of length M).
 *   mode MLS_MODE_PAPER (eq. (3) summed over sub-models):
 *     student g_ce = w (1 - alpha), g_kl = w alpha tau^2; teacher g_ce = w, g_kl = 0
 *   mode MLS_MODE_ADDITIVE:
 *     student g_ce = w, g_kl = w alpha tau^2; teacher g_ce = w, g_kl = 0
 * w is the per-sub-model loss weight (appendix G); NULL means all ones.
 */
mls_status mls_coeffs(int32_t M, int32_t teacher, float alpha, float tau, int32_t mode,
                      const float* w, float* g_ce, float* g_kl);

/* Reads the device flags (mls_device_flags) and the valid-token count from a
 * statistics buffer. Synchronises the stream. Either output may be NULL. */
mls_status mls_read_stats_header(const mls_problem* p, const void* stats, void* stream,
                                 int32_t* n_valid, int32_t* device_flags);

/*
 * Device-side errors of the forward pass (paper section 2, eq. (2) and
 * eq. (3) need finite logits and labels in [0, V)): *flags receives the OR of
 * mls_device_flags the last mls_distill_fwd (or mls_distill_fwd_bwd) on this
 * statistics buffer raised: MLS_DEVFLAG_LABEL_RANGE for a label outside
 * [0, V) that is not ignore_index, MLS_DEVFLAG_NONFINITE for a NaN or
 * infinite per-token statistic of a valid token. The flags live in the
 * statistics buffer's header (the forward rewrites them on every call), so
 * calls on different buffers do not interfere. Waits for the stream: call it
 * after the forward, not inside a timed or captured region.
 */
mls_status mls_device_error(const mls_problem* p, const void* stats, void* stream, int32_t* flags);

/*
 * Kernel timing, a tracing aid for benchmarks. While enabled (per calling
 * thread), every kernel the library enqueues from that thread is bracketed
 * by two hipEvents recorded on the same stream. mls_profile_report waits for
 * the recorded events, writes at most max_entries aggregated rows (one per
 * kernel name, in first-launch order) and clears the record.
 */
typedef struct mls_kernel_time {
  char name[32];
  int32_t launches;
  double total_ms;
} mls_kernel_time;

mls_status mls_profile_enable(int32_t enable);
mls_status mls_profile_report(mls_kernel_time* out, int32_t max_entries, int32_t* n_out);

/*
 * Measurement aid: the MFMA ceiling of the device. Enqueues one launch in which
 * every wave issues iters x 8 independent v_mfma_f32_32x32x16_bf16 on operands
 * held in registers (no memory or LDS traffic): all-zero operands, or random
 * bf16 values when random_operands is nonzero (the clock responds to the data's
 * switching activity). *flops receives the launch's floating-point operations
 * (divide by its duration for the rate). sink: device float32 array of at least
 * 524288 entries that receives per-thread sums (it keeps the work live); with
 * sink NULL only *flops is written. Asynchronous on stream.
 */
mls_status mls_mfma_probe(int32_t random_operands, int32_t iters, float* sink, size_t sink_floats,
                          double* flops, void* stream);

/* Static text for a status code. */
const char* mls_status_string(mls_status s);

/* Detail of the last error returned on the calling thread ("" if none). */
const char* mls_last_error(void);

/* Library version string. */
const char* mls_version(void);

/*
 * Host helper: properties of the current device that set its nominal peaks
 * (compute units, peak engine clock in kHz, peak memory clock in kHz, memory
 * bus width in bits; from hipDeviceGetAttribute). Any output may be NULL.
 * The bf16 dense MFMA peak of a gfx950 part is CUs x clock x 4096 FLOP per
 * clock per CU.
 */
mls_status mls_device_info(int32_t* compute_units, int32_t* clock_khz, int32_t* mem_clock_khz,
                           int32_t* mem_bus_bits);

#ifdef __cplusplus
}
#endif

#endif /* MLS_H_ */
