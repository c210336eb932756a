/*
 * ssd.h — C ABI of the self-speculative decoding library (FastVLM, arXiv 2510.22641) for
 * MI355X (gfx950).
 *
 * The paper's inference problem (Algorithm 1, Sec. "Methodology", paragraph "Inference"): given
 * the encoder output z = E(I, T0), a context y^1..y^t, a target length T and a draft length d,
 * generate tokens with a draft model (the decoder's first n layers, the imitation network I and
 * the shared LM head g) that proposes d tokens autoregressively, and the full decoder, which
 * verifies them in one forward pass; the longest agreeing prefix is kept together with the full
 * model's token at the first disagreement (or its next token when all agree).  Draft and full
 * model share one KV cache (Sec. "Methodology", paragraph "KV cache").
 *
 * This library computes the four steps of that loop on the GPU:
 *   ssd_prefill  run the full decoder over the context, fill the KV cache, emit the first token
 *   ssd_draft    gamma draft steps (layers 1..k, I, g, argmax) from the pending token
 *   ssd_verify   the full decoder over [pending, draft_1..draft_gamma] in one causal pass
 *   ssd_accept   greedy acceptance; advances the valid KV length (the rollback is the reset)
 * and, for convenience, the whole loop (ssd_generate).
 *
 * Conventions
 *   - Every pointer named d_* (and every pointer inside ssd_weights / ssd_kv) is device memory
 *     owned by the caller, which keeps it alive until the stream has finished the work.  The
 *     library allocates no device memory; it uses the caller's workspace (ssd_workspace_bytes).
 *   - Matrices are row-major [out][in] (y = W x).  Matrices, embeddings and visual tokens are
 *     in `wdtype`; norm gains, imitation-network biases and the relative-position bias table are
 *     float32.  KV pools are in `kvdtype`.
 *   - All calls are asynchronous on the stream given to ssd_create, except ssd_sync_status and
 *     ssd_generate, which synchronise it.  One context per stream; not thread-safe.
 *   - Return value: SSD_OK (0) or a negative SSD_ERR_* code; nothing is launched on error.
 *     Faults detected on the device (token id out of range, position beyond the KV capacity,
 *     page id out of range) set bits in a device status word that ssd_sync_status reports;
 *     the offending access is skipped, never performed.
 */
#ifndef SSD_H
#define SSD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  SSD_OK = 0,
  SSD_ERR_ARG = -1,      /* null pointer or a value out of range                         */
  SSD_ERR_SHAPE = -2,    /* B > max_batch, gamma > max_gamma, unsupported dimensions       */
  SSD_ERR_CAPACITY = -3, /* context or workspace too small                                 */
  SSD_ERR_HIP = -4,      /* a HIP runtime call or kernel launch failed                      */
  SSD_ERR_STATE = -5,    /* call out of order (draft/verify before prefill, stale reuse)   */
  SSD_ERR_DEVICE = -6    /* ssd_sync_status: the device status word is non-zero           */
};

enum { SSD_ARCH_T5 = 0, SSD_ARCH_LLAMA = 1 };
enum { SSD_F32 = 0, SSD_BF16 = 1 };
enum {
  SSD_MODE_GREEDY = 0,
  SSD_MODE_SPECULATIVE = 1,
  SSD_MODE_SPECULATIVE_DYNAMIC = 2
};

/* device status bits (ssd_sync_status; ssd_generate returns SSD_ERR_DEVICE when one is set) */
enum { SSD_DEV_BAD_TOKEN = 1, SSD_DEV_CAPACITY = 2, SSD_DEV_BAD_PAGE = 4 };

/* Decoder and context dimensions, copied at ssd_create. */
typedef struct {
  int32_t arch;         /* SSD_ARCH_T5: RMSNorm, self-attn + T5 relative bias, cross-attn to z,
                           gated-GELU FFN; SSD_ARCH_LLAMA: RMSNorm, RoPE self-attn, SwiGLU */
  int32_t n_layers;     /* L */
  int32_t d_model;      /* d, multiple of 64 */
  int32_t n_heads;      /* H */
  int32_t d_head;       /* 64 or 128 */
  int32_t d_ff;         /* multiple of 64 */
  int32_t vocab;        /* V */
  int32_t n_visual;     /* T5: visual tokens attended by cross-attention; LLaMA: prefix rows */
  int32_t rel_buckets;  /* T5 relative-position buckets (32) */
  int32_t rel_max_dist; /* T5 bucket max distance (128) */
  float rope_theta;     /* LLaMA rotary base (10000) */
  float norm_eps;       /* decoder RMSNorm eps (T5 1e-6, LLaMA 1e-5) */
  float ln_eps;         /* imitation-network LayerNorm eps (1e-5) */
  int32_t wdtype;       /* SSD_F32 or SSD_BF16: matrices, embeddings, visual tokens */
  int32_t kvdtype;      /* SSD_F32 or SSD_BF16: KV pools and cross-attention K/V */
  int32_t draft_layers; /* k: the draft model is layers 1..k + imitation network + LM head */
  int32_t in_hidden;    /* imitation-network hidden width (multiple of 64) */
  int32_t in_residual;  /* 1: I(x) = x + FC2(GELU(FC1(LN(x)))); 0: FC2(GELU(FC1(LN(x)))) */
  int32_t max_batch;    /* B capacity */
  int32_t max_gamma;    /* largest draft length used with this context */
  int32_t max_seq;      /* KV positions per sequence: prefix + prompt + T + max_gamma + 1; with the
                           stepwise calls on a batch whose sequences finish in different rounds,
                           max_gamma more (a finished sequence is still drafted and verified at
                           its last length until the batch is done) */
  int32_t max_prompt;   /* largest prompt length P passed to ssd_prefill */
  int32_t page_size;    /* KV positions per page */
  int32_t max_pages;    /* page-table columns per sequence (>= ceil(max_seq / page_size)) */
} ssd_dims;

/* Per-layer weights (device pointers).  HD = n_heads * d_head. */
typedef struct {
  const float* attn_norm; /* [d] */
  const void* wq;         /* [HD][d] */
  const void* wk;         /* [HD][d] */
  const void* wv;         /* [HD][d] */
  const void* wo;         /* [d][HD] */
  const float* xattn_norm;/* [d]      T5 only (NULL for LLaMA) */
  const void* xq;         /* [HD][d]  T5 only */
  const void* xk;         /* [HD][d]  T5 only: applied to z at prefill */
  const void* xv;         /* [HD][d]  T5 only: applied to z at prefill */
  const void* xo;         /* [d][HD]  T5 only */
  const float* ffn_norm;  /* [d] */
  const void* w_gate;     /* [d_ff][d] */
  const void* w_up;       /* [d_ff][d] */
  const void* w_down;     /* [d][d_ff] */
} ssd_layer_weights;

typedef struct {
  const void* embed;      /* [V][d] */
  const void* lm_head;    /* [V][d]  g = final RMSNorm then this matrix (shared by draft and full) */
  const float* final_norm;/* [d] */
  const float* rel_bias;  /* [rel_buckets][H]  T5 only */
  const float* in_ln_w;   /* [d]  imitation network: LayerNorm gain */
  const float* in_ln_b;   /* [d]  LayerNorm shift */
  const void* in_w1;      /* [in_hidden][d] */
  const float* in_b1;     /* [in_hidden] */
  const void* in_w2;      /* [d][in_hidden] */
  const float* in_b2;     /* [d] */
  const ssd_layer_weights* layers; /* host array of n_layers entries (copied at ssd_create) */
} ssd_weights;

/* The shared KV cache (device pointers, caller-owned). */
typedef struct {
  void* k_pool;              /* [L][n_pages][H][page_size][d_head] kvdtype */
  void* v_pool;              /* same layout */
  int32_t n_pages;           /* pages per layer in the pools */
  const int32_t* page_table; /* [max_batch][max_pages]: page of positions [j*page_size, (j+1)*page_size) */
  int32_t* seq_len;          /* [max_batch]: valid positions; written only by prefill and accept */
  void* xk;                  /* T5: [L][max_batch][H][n_visual][d_head] kvdtype, written by prefill */
  void* xv;                  /* T5: same */
} ssd_kv;

typedef struct ssd_ctx ssd_ctx;

/* Workspace bytes a context with these dimensions needs (0 if the dimensions are invalid): the
 * residual rows, the staged layer-k states, the operand planes of the MFMA paths, argmax and
 * attention partials, the bias / rotary tables, the folded T5 cross-attention of a one-sequence
 * context, and, when a context block can exceed 128 rows, four float32 K-range partials of the
 * prefill's residual projections. */
size_t ssd_workspace_bytes(const ssd_dims* dims);

/* Validate dimensions, copy the weight and KV descriptors, carve the workspace and build the
 * relative-bias (T5) or rotary (LLaMA) tables into it.  `stream` is a hipStream_t (NULL: the
 * null stream).  On success *out receives a host-side context that ssd_destroy frees. */
int ssd_create(const ssd_dims* dims, const ssd_weights* w, const ssd_kv* kv, void* d_workspace,
               size_t workspace_bytes, void* stream, ssd_ctx** out);

/* For callers that cannot allocate device memory (code running under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): ssd_create without a workspace argument.  The
 * context's workspace is the library's own fixed device array of SSD_STATIC_SCRATCH_BYTES
 * (64 MiB), one per GPU, which each GPU the library runs on holds until the process ends; it is
 * the array of the device current at the call (that of `stream`).  Everything else is as
 * ssd_create, except that:
 *   - the T5 cross-attention is not folded (its per-layer float32 matrices would not fit), so
 *     one-row steps take the query projection, attention and output projection instead (the
 *     same decoder, within the same parity tolerances);
 *   - HIP graphs are off (instantiating one allocates); ssd_set_graphs(ctx, 1) turns them on,
 *     and then the first call of each shape allocates its graph;
 *   - ssd_generate's read-back goes to host stack memory instead of a pinned buffer.
 * Neither this call nor any later call on the context calls hipMalloc, hipHostMalloc, hipFree or
 * another allocating routine, on the device or the host.  Dimensions whose workspace
 * (ssd_workspace_bytes without the folded matrices) exceeds SSD_STATIC_SCRATCH_BYTES are refused
 * with SSD_ERR_CAPACITY before anything runs.  At most one such context per device is alive at a
 * time (a second call before ssd_destroy of the first returns SSD_ERR_STATE): every context made
 * here on one GPU shares that GPU's array, which keeps the previous context's contents (this
 * call rebuilds the tables and clears the status word; every other slice is written before it
 * is read), and work of two of them that overlapped on one GPU would race. */
#define SSD_STATIC_SCRATCH_BYTES ((size_t)64 << 20)
int ssd_create_static(const ssd_dims* dims, const ssd_weights* w, const ssd_kv* kv, void* stream,
                      ssd_ctx** out);

/* Prefill (Algorithm 1's input: z and the context y^1..y^t).  d_prompt [B][P] int32 token ids;
 * d_visual [B][n_visual][d] wdtype.  T5: cross-attention K/V of every layer are projected from
 * z; the prompt occupies positions 0..P-1.  LLaMA: the visual rows are the inputs of positions
 * 0..n_visual-1, the prompt follows.  Sets seq_len[b] to the context length and writes the full
 * model's argmax at the last context position to d_pending[b] (emitted token #1).
 * d_logits [B][V] float32 receives those logits when not NULL.  For a one-sequence T5 context
 * the folded cross-attention of every layer is formed on a second stream of the context
 * (created at the first prefill, default priority) beside the prompt's own pass; the context's
 * stream waits for it before the call's work ends, so stream order holds for the caller. */
int ssd_prefill(ssd_ctx* ctx, int B, int P, const int32_t* d_prompt, const void* d_visual,
                int32_t* d_pending, float* d_logits);

/* Drafting stage (Algorithm 1, draft loop): for i = 0..gamma-1 run layers 1..k, the imitation
 * network and g at position seq_len[b]+i on u_i (u_0 = d_pending[b], u_{i+1} = the draft's
 * argmax), writing layer 1..k KV there.  d_draft [B][gamma] int32; d_draft_logits
 * [B][gamma][V] float32 or NULL.  Keeps each step's layer-k hidden state for ssd_verify's reuse.
 * Does not change seq_len.  1 <= gamma <= max_gamma. */
int ssd_draft(ssd_ctx* ctx, int B, int gamma, const int32_t* d_pending, int32_t* d_draft,
              float* d_draft_logits);

/* Verification stage (Algorithm 1, verify loop): the full decoder over u_0..u_gamma =
 * [d_pending[b], d_draft[b][0..gamma-1]] at positions seq_len[b]..seq_len[b]+gamma in one causal
 * pass, writing KV of every layer there.  d_target [B][gamma+1] int32 receives the full model's
 * argmax at each of those positions; d_logits [B][gamma+1][V] float32 or NULL.
 * reuse_hidden = 1 takes layers 1..k of positions 0..gamma-1 from the immediately preceding
 * ssd_draft (same B, gamma and inputs) and runs them only for the last position; 0 recomputes.
 * gamma = 0 is one full-model greedy step.  Does not change seq_len.  d_draft may hold any
 * tokens (e.g. forced from the host). */
int ssd_verify(ssd_ctx* ctx, int B, int gamma, const int32_t* d_pending, const int32_t* d_draft,
               int reuse_hidden, int32_t* d_target, float* d_logits);

/* Greedy acceptance (Algorithm 1, verify loop): a[b] = the number of leading i with
 * draft[b][i] == target[b][i]; d_out[b][0..a] = draft[b][0..a-1], target[b][a]; d_accept_len[b] =
 * a; seq_len[b] += a + 1 (KV beyond it is stale and never read); d_pending[b] = target[b][a].
 * Sequences with d_active[b] == 0 are left untouched (d_active may be NULL: all active). */
int ssd_accept(ssd_ctx* ctx, int B, int gamma, const int32_t* d_draft, const int32_t* d_target,
               int32_t* d_pending, int32_t* d_out, int32_t* d_accept_len, const int32_t* d_active);

/* Sampling variant of the loop (speculative sampling; the paper's decoder may sample its next
 * token instead of taking the argmax, Sec. "SSD Setup for VLMs").  Distributions at temperature
 * `temperature` (> 0): softmax(logits / temperature).  Randomness is an input: a sample from
 * weights w with uniform u in [0, 1) is the inverse CDF, the smallest k with
 * w_0 + ... + w_k > u * sum(w).
 *
 * ssd_draft_sample: ssd_draft with each draft token sampled from the draft's distribution
 * (d_u [B][gamma]: the uniform of step i of sequence b at [b][i]); d_draft_logits
 * [B][gamma][V] float32 is required (the acceptance needs it).  A following ssd_verify may reuse
 * the layer-k states as after ssd_draft.
 *
 * ssd_accept_sample: the speculative-sampling rule on the drafts of ssd_draft_sample and the
 * full model's logits from ssd_verify (d_target_logits [B][gamma+1][V], required).  Draft i is
 * accepted when u[b][i] * q_i(draft_i) < p_i(draft_i), q_i the draft's and p_i the full model's
 * distribution at the same position (probability min(1, p/q)); the first rejected position
 * emits a sample from the normalised residual max(0, p_i - q_i) (p_i if it vanishes) drawn with
 * u[b][gamma], and a round whose drafts all pass emits a sample from p_gamma drawn with
 * u[b][gamma] (d_u [B][gamma + 1]).  Outputs as ssd_accept: d_out[b][0..a] = the a accepted
 * drafts and the sampled token, d_accept_len[b] = a, seq_len[b] += a + 1, d_pending[b] = the
 * sampled token; sequences with d_active[b] == 0 are left untouched.  The output sequence then
 * follows the full model's sampling distribution. */
int ssd_draft_sample(ssd_ctx* ctx, int B, int gamma, const int32_t* d_pending, const float* d_u,
                     float temperature, int32_t* d_draft, float* d_draft_logits);
int ssd_accept_sample(ssd_ctx* ctx, int B, int gamma, const int32_t* d_draft,
                      const float* d_draft_logits, const float* d_target_logits, const float* d_u,
                      float temperature, int32_t* d_pending, int32_t* d_out,
                      int32_t* d_accept_len, const int32_t* d_active);

/* Confidence-stopped drafting, the rule of Draft & Verify, the self-speculative baseline the
 * paper compares with (Sec. "Experiments", baselines: drafting halts once the draft's confidence
 * drops below a threshold).  The confidence of a draft is its largest softmax probability,
 * max_v softmax(draft logits)_v (the paper's confidence C_l, appendix on the choice of n).
 *
 * ssd_draft_confident: ssd_draft, except that sequence b stops drafting after the first step
 * whose confidence is below `threshold` (that step's token is still proposed), so it proposes
 * d_ndraft[b] in [1, gamma] drafts (0 for a sequence with d_active[b] == 0; d_active may be
 * NULL: all active).  Steps run while an active sequence still drafts: after every step but the
 * last the stream is synchronised and the flags read back (not when threshold <= 0, where no
 * sequence stops); *h_steps (host) receives the steps run, the largest d_ndraft.  d_draft
 * receives [B][*h_steps] (row stride *h_steps; entries past d_ndraft[b] are the draft model's
 * further tokens, not proposals); d_conf [B][gamma] float32 or NULL receives each step's
 * confidence, d_draft_logits [B][gamma][V] or NULL the logits.  A following ssd_verify with
 * gamma = *h_steps and the same d_pending / d_draft may reuse the layer-k states.
 *
 * ssd_accept_counts: ssd_accept with sequence b's acceptance limited to its d_ndraft[b] drafts
 * (a[b] <= d_ndraft[b]; the emitted token at a[b] is target[b][a[b]]).
 *
 * ssd_generate_confident: ssd_generate (SSD_MODE_SPECULATIVE, gamma drafts at most) with
 * confidence-stopped drafting at `threshold`; the stream is synchronised once per round and
 * after each draft step as above; h_stats counts the drafts proposed. */
int ssd_draft_confident(ssd_ctx* ctx, int B, int gamma, float threshold, const int32_t* d_pending,
                        const int32_t* d_active, int32_t* d_draft, int32_t* d_ndraft,
                        float* d_conf, float* d_draft_logits, int* h_steps);
int ssd_accept_counts(ssd_ctx* ctx, int B, int gamma, const int32_t* d_draft,
                      const int32_t* d_ndraft, const int32_t* d_target, int32_t* d_pending,
                      int32_t* d_out, int32_t* d_accept_len, const int32_t* d_active);
int ssd_generate_confident(ssd_ctx* ctx, int B, int P, const int32_t* d_prompt,
                           const void* d_visual, int T, int gamma, float threshold,
                           int reuse_hidden, int32_t* d_tokens, int64_t* h_stats);

/* The whole loop: prefill, then rounds of draft + verify + accept (SSD_MODE_SPECULATIVE) or
 * verify(gamma = 0) + accept (SSD_MODE_GREEDY) until T tokens per sequence are emitted (the last
 * round truncated; a finished sequence's seq_len then counts only the positions it emitted, so
 * max_seq = prefix + prompt + T + max_gamma + 1 suffices for any batch).  d_tokens [B][T] int32.
 * SSD_MODE_SPECULATIVE_DYNAMIC drafts ssd_dynamic_gamma(t, gamma, max_seq) tokens per round
 * (appendix on the choice of d: d grows with the context length t), t = the shortest context
 * length among the sequences still active at the start of the round; gamma + 9 <= max_gamma.
 * h_stats (host, may be NULL) receives {rounds, sum over sequences of accepted drafts, sum of
 * drafted tokens}.  Synchronises the stream to test for completion: with a fixed gamma (and in
 * greedy mode) once per batch of rounds, a batch being the ceil(L / (gamma + 1)) rounds that are
 * certainly needed (L: the most tokens a sequence still active lacks); in the dynamic mode once
 * per round.  Each of these read-backs also carries the device status word: when it is non-zero
 * (a bad token id, a position past the cache, an unmapped page), no further round is launched and
 * SSD_ERR_DEVICE is returned, as it is when the word is set after the last round; the word is
 * left set for ssd_sync_status to report and clear. */
int ssd_generate(ssd_ctx* ctx, int B, int P, const int32_t* d_prompt, const void* d_visual, int T,
                 int gamma, int mode, int reuse_hidden, int32_t* d_tokens, int64_t* h_stats);

/* Draft length at context length t (appendix on the choice of d): d0 + floor(10 * sigmoid(0.01 *
 * (t - n_max / 2))); n_max is the maximum sequence length.  In [d0, d0 + 9] for 0 <= t <= n_max
 * (d0 + 10 only where the double-precision logistic rounds to 1).  Host function. */
int ssd_dynamic_gamma(int t, int d0, int n_max);

/* Capture ssd_draft / ssd_verify launch sequences into HIP graphs and replay them (1, default)
 * or launch kernels one by one (0). */
int ssd_set_graphs(ssd_ctx* ctx, int enable);

/* Hidden-state export, for fitting the imitation network offline on the decoder's own states
 * (a stand-in for the paper's imitation training, Sec. "Deep Representation Imitation"; not on
 * the decode path).  While set (all three non-NULL), every ssd_draft also copies, for its
 * gamma steps, the imitation network's hidden features gelu(W1 LN(x_k) + b1) to
 * d_phi [B][gamma][in_hidden] and the layer-k residual rows x_k to d_xk [B][gamma][d_model], and
 * every ssd_verify copies its final residual rows (after the last layer, before g's norm) to
 * d_xl [B][gamma + 1][d_model], float32, device memory owned by the caller (sized for the
 * largest B and gamma used).  Row i of a draft and row i of the verify that follows it are the
 * same position.  All NULL disables; a mix of NULL and non-NULL is SSD_ERR_ARG. */
int ssd_set_hidden_export(ssd_ctx* ctx, float* d_phi, float* d_xk, float* d_xl);

/* Kernel timing for roofline reports.  While enabled (and graphs are bypassed), every launch of
 * the one-row weight-streaming GEMV that streams the RMS-normalised d_model-wide matrices (QKV,
 * cross-attention query, gate/up, LM head; the kernel that carries most of a batch-1 draft step:
 * gemv1k_kernel<unsigned short, KP, 1> with KP = ceil(d_model / 2048) for bf16 weights and
 * 2048 <= d_model <= 6144, else gemv1_kernel<T, KP, 1> with KP = 2 for d_model <= 1024, 4 for
 * d_model <= 2048, 12 for 4096 < d_model <= 6144, else 8) is launched with two HIP events bound to its own dispatch on
 * the context's stream, so their elapsed time is the kernel's execution time; its algorithmic
 * bytes (weights + input row + output row) are added up.  ssd_profile_read synchronises the stream and returns
 * the number of such launches, the summed kernel time in seconds and the summed bytes since the
 * previous read (any pointer may be NULL).  Costs one event pair per launch; for measurement only. */
int ssd_profile_enable(ssd_ctx* ctx, int enable);
int ssd_profile_read(ssd_ctx* ctx, int64_t* launches, double* seconds, double* bytes);

/* Measurement utility, not on the decode path: the HBM read ceiling the kernels' byte rates are
 * compared with.  Streams `bytes` (a multiple of 16; use far more than the 256 MB Infinity Cache)
 * of device memory at d_buf through a read-only kernel (one 16 KB chunk per block of 256
 * threads, 16-byte loads, four in flight per thread) reps + 1 times on `stream`, the first pass
 * a warm-up, and returns the best rate in GB/s (HIP events around each pass) in *gbps.  d_out
 * (4096 floats) is a sink the kernel may write.  Synchronises the stream. */
int ssd_read_bandwidth(const void* d_buf, size_t bytes, float* d_out, int reps, void* stream,
                       double* gbps);

/* Synchronise the stream; SSD_OK, SSD_ERR_HIP, or SSD_ERR_DEVICE when the device status word is
 * non-zero (then *status, if not NULL, receives the SSD_DEV_* bits) — and clear the word. */
int ssd_sync_status(ssd_ctx* ctx, int32_t* status);

/* Human-readable name of a return code. */
const char* ssd_status_string(int code);

/* Free the host-side context (device buffers belong to the caller). */
void ssd_destroy(ssd_ctx* ctx);

#ifdef __cplusplus
}
#endif

#endif /* SSD_H */
