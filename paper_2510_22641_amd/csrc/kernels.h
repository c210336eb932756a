// Host-side launch interface of the gfx950 kernels (internal to libssd).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ssd.h"

typedef uint16_t bf16_t;

namespace ssd {

// Input transform of a linear layer: none, RMSNorm (gain), LayerNorm (gain, shift), or a softmax
// over consecutive groups of LinearArgs::group inputs (the folded cross-attention's probabilities;
// one-row vector path only).
enum Norm { NORM_NONE = 0, NORM_RMS = 1, NORM_LN = 2, NORM_SOFTMAX = 3 };

// Paged KV addressing shared by the QKV epilogue and the attention kernels.
struct PagedKV {
  void* k;  // layer base of the pools [n_pages][H][page_size][dh]
  void* v;
  const int32_t* page_table;
  int max_pages;
  int page_size;
  int n_pages;
  const int32_t* seq_len;
  int pos_off;  // row j of sequence b sits at position seq_len[b] + pos_off + j
};

enum Epi {
  EPI_STORE = 0,       // y[m][n] = acc
  EPI_RESID = 1,       // y[m][n] += acc  (and stash[m][n] = y[m][n] when stash != null)
  EPI_GATED_GELU = 2,  // y[m][n] = gelu_tanh(acc_gate) * acc_up  (w[0] = gate, w[1] = up)
  EPI_GATED_SILU = 3,  // y[m][n] = silu(acc_gate) * acc_up
  EPI_BIAS_GELU = 4,   // y[m][n] = gelu_tanh(acc + bias[n])
  EPI_BIAS_RESID = 5,  // y[m][n] = (resid ? resid[m][n] : 0) + acc + (bias ? bias[n] : 0)
  EPI_ARGMAX = 6,      // per-block (max, argmax) over n for each m; logits[m][n] = acc if wanted
  EPI_QKV = 7          // w = (wq, wk, wv): rotary on q and k (when rope_cos is set), q -> y[m][.],
                       // k and v into the paged pools at the row's position (vector path only)
};

// y = epilogue( W . norm(x) ) for M rows.  The output features are up to three matrices of
// n_per rows each, concatenated (QKV), or the pair (gate, up) for the gated epilogues.
struct LinearArgs {
  const float* x = nullptr;  // [M][ldx] float32 inputs
  int ldx = 0;
  int M = 0;
  int K = 0;
  int norm = NORM_NONE;
  const float* gain = nullptr;
  const float* shift = nullptr;
  float eps = 0.f;
  int group = 0;  // NORM_SOFTMAX: inputs per softmax group (8, 16, 32 or 64)
  // NORM_SOFTMAX (one-row path): when set, the inputs are first multiplied by
  // 1 / sqrt(mean(pre_row[0..pre_len)^2) + eps) (the RMS normalisation of the row the scores were
  // projected from); 4 <= pre_len <= 2048, a multiple of 4
  const float* pre_row = nullptr;
  int pre_len = 0;
  const void* w[3] = {nullptr, nullptr, nullptr};  // [n_per][K] each, wdtype
  int n_mats = 1;
  int n_per = 0;
  int wdtype = 0;  // 0 f32, 1 bf16
  int epi = EPI_STORE;
  float* y = nullptr;
  int ldy = 0;
  const float* bias = nullptr;
  const float* resid = nullptr;
  int ldr = 0;
  float* stash = nullptr;
  int lds = 0;
  // EPI_ARGMAX
  float* part_val = nullptr;  // [M][n_parts]
  int* part_idx = nullptr;
  int n_parts = 0;            // filled by argmax_parts()
  float* logits = nullptr;    // [M][ldl] or null
  int ldl = 0;
  // EPI_QKV: row m = b*C + j sits at position kv.seq_len[b] + kv.pos_off + j
  PagedKV kv = {};
  int C = 1, n_heads = 0, d_head = 0, kvdtype = 0, max_seq = 0;
  const float* rope_cos = nullptr;  // [max_seq][d_head/2] or null (no rotation)
  const float* rope_sin = nullptr;
  int32_t* status = nullptr;        // SSD_DEV_CAPACITY / SSD_DEV_BAD_PAGE bits
  // row statistics for the MFMA path's normalisation (filled by launch_linear)
  float2* stats = nullptr;    // [M] workspace
  int use_mfma = -1;          // -1: choose; 0: vector path; 1: MFMA path
  // Skinny path operands, in buffers of plane_rows rows (a multiple of 16, >= M).  Input: bf16
  // planes hi / lo of the (gain-multiplied) rows, hi row m at in_planes + m * in_ld, lo row m at
  // in_planes + (plane_rows + m) * in_ld; with NORM_RMS, 1/rms of row m comes from the partial sums
  // of squares in_ssq[p * plane_rows + m], p < in_nssq.
  int plane_rows = 16;
  const bf16_t* in_planes = nullptr;
  int in_ld = 0;
  const float* in_ssq = nullptr;
  int in_nssq = 0;
  // launch_linear_skinny_fold with NORM_SOFTMAX: float32 input rows (row m at in_f32 + m * in_ld)
  // turned into softmax probabilities over groups of `group` consecutive inputs.
  const float* in_f32 = nullptr;
  // Output planes for the next skinny launch (EPI_RESID: of out_gain * y_new, plus per-block
  // partial sums of squares of y_new in out_ssq[block * plane_rows + m]; gated: of y; null: none).
  bf16_t* out_planes = nullptr;
  int out_ld = 0;
  float* out_ssq = nullptr;
  const float* out_gain = nullptr;
  // Tile path (rows past the skinny capacity): a buffer for the bf16 hi / lo planes of the
  // (gain-multiplied) input rows, gemm_plane_rows rows of at most gemm_plane_ld elements per
  // plane; null keeps the tile kernels that split the inputs themselves.
  bf16_t* gemm_planes = nullptr;
  int gemm_plane_rows = 0;
  int gemm_plane_ld = 0;
  // Tile path, residual projections (y += W . x): partial products over ranges of K, float32
  // [kpart_max][gemm_plane_rows][kpart_ld], which a second launch adds to y in range order; null
  // keeps one pass over K.  ksplit is set by the launcher.
  float* kpart = nullptr;
  int kpart_max = 0;
  int kpart_ld = 0;
  int ksplit = 1;
};

// Kernel-level timing of the one-row GEMV launches with K inputs, input normalisation `norm` and
// weight type `wdtype` (gemv1k_kernel for bf16 rows of 2048..6144, else gemv1_kernel): when start / stop are set and
// the launch is one of those, it is launched with the events bound to its own dispatch
// (hipExtLaunchKernel), so their elapsed time is the kernel's execution time; `timed` reports
// whether it happened.
struct LaunchTiming {
  hipEvent_t start = nullptr, stop = nullptr;
  int K = 0;
  int norm = NORM_RMS;
  int wdtype = 1;
  bool timed = false;
};

// Pieces per batch (the KP of gemv_kernel) the vector path uses for rows of K elements.
int gemv_pieces(int K);

// Launch y = epilogue(W . norm(x)).  For EPI_ARGMAX, *n_parts receives the number of partials
// per row written to part_val / part_idx (their row stride).
hipError_t launch_linear(LinearArgs a, hipStream_t s, int* n_parts = nullptr,
                         LaunchTiming* timing = nullptr);

// Two one-row GEMVs that read the same inputs, in one launch (the blocks of `a` first, then those
// of `b`): `a` with bf16 weights and K <= 2048, `b` with float32 weights and K <= 4096, no input
// transform, store / residual / bias epilogues only.
bool linear_pair_ok(const LinearArgs& a, const LinearArgs& b);
hipError_t launch_linear_pair(const LinearArgs& a, const LinearArgs& b, hipStream_t s);

// Upper bound of the partials per row for n_out outputs (workspace sizing).
int argmax_parts_max(int n_out);

// Rows of a verify chunk (2..128, bf16 weights) take the skinny MFMA path (16 rows per block
// row of the grid): the inputs arrive as bf16 planes written once by their producer (a.in_planes
// ..., see LinearArgs), with RMSNorm folded (a.norm = NORM_RMS: the gain is already in the planes,
// 1/rms from a.in_ssq) or none; the gated, QKV (rotary + KV store), residual (+ next planes), bias
// and argmax epilogues.
bool skinny_ok(int M, int K, int wdtype);
hipError_t launch_linear_skinny(const LinearArgs& a, hipStream_t s, int* n_parts = nullptr);

// Planes of gain * x for M <= plane_rows rows (hi row m at out + m * ldo, lo at
// out + (plane_rows + m) * ldo) and the full-row sums of squares ssq[m] (one partial): the input
// of the first skinny launch of a pass.
hipError_t launch_skinny_prep(const float* x, int ldx, int M, int K, const float* gain,
                              bf16_t* out, int ldo, int plane_rows, float* ssq, hipStream_t s);

// 16-feature tiles of a skinny launch.
int skinny_blocks(int n_out);
// The folded cross-attention of a verify chunk (at most 8 rows, float32 weights) on half tiles:
// the scores fold_q . rms(x) (NORM_RMS, EPI_STORE, input planes as launch_linear_skinny's) or the
// output y += fold_o . softmax(scores) per group (NORM_SOFTMAX, EPI_RESID, float32 input rows
// in_f32).  skinny_fold_ok tells whether a chunk of M rows with these sizes takes this path.
bool skinny_fold_ok(int d_model, int n_fold, int group, int M);
hipError_t launch_linear_skinny_fold(const LinearArgs& a, hipStream_t s);
// Partial sums of squares a skinny residual epilogue of n_out features over M rows leaves (the
// in_nssq of its consumer): one per tile, or two with half tiles.
int skinny_ssq_parts(int n_out, int M);

// True when launch_linear takes the weight-streaming vector path (the one that has EPI_QKV).
bool linear_is_vector(const LinearArgs& a);

// Algorithmic HBM bytes of a launch: weights + input rows + output rows (+ residual reads).
double linear_bytes(const LinearArgs& a);

// Gather input rows: x[r] = embedding of a token or a visual row.
// Row r = b*C + j; j < n_prefix: visual[b][j]; else token = t0[b] if (t0 && j' == 0) else
// t1[b*ld1 + j' - (t0 ? 1 : 0)] with j' = j - n_prefix.
struct EmbedArgs {
  float* x;
  int B, C, d;
  const void* embed;
  int vocab;
  int wdtype;
  const int32_t* t0;
  const int32_t* t1;
  int ld1;
  const void* visual;  // [B][n_visual][d] wdtype
  int n_visual;
  int n_prefix;
  int32_t* status;
};
hipError_t launch_embed(const EmbedArgs& a, hipStream_t s);

// q/k/v rows (qkv [R][3*HD], R = B*C) -> rotary (LLaMA) -> q_out [R][HD], K/V into the pools.
struct RopeScatterArgs {
  const float* qkv;
  float* q_out;
  int B, C, H, dh;
  int kvdtype;
  PagedKV kv;
  const float* rope_cos;  // [max_seq][dh/2] or null (no rotation)
  const float* rope_sin;
  int max_seq;
  int32_t* status;
};
hipError_t launch_rope_scatter(const RopeScatterArgs& a, hipStream_t s);

constexpr int ATTN_SPLITS_MAX = 8;

struct AttnArgs {
  const float* q;  // [B*C][H*dh]
  float* out;      // [B*C][H*dh]
  bf16_t* out_planes = nullptr;  // optional hi / lo bf16 planes of out (lo plane_rows rows on)
  int plane_rows = 16;
  // key-split partials (long contexts): [part_rows][H][ATTN_SPLITS_MAX][dh + 2] floats, or null
  float* part = nullptr;
  int part_rows = 0;
  int B, C, H, dh;
  int kvdtype;
  int cross;         // 0: causal over the paged cache; 1: dense over n_keys cross-attention keys
  PagedKV kv;        // self-attention
  const float* bias; // [H][max_seq] by distance (T5 self-attention) or null
  int max_seq;
  const void* xk;    // cross: [B][H][n_keys][dh]
  const void* xv;
  int n_keys;
  float scale;
  int32_t* status;
};
hipError_t launch_attention(const AttnArgs& a, hipStream_t s);

// Cross-attention of one sequence folded into two float32 matrices per layer (T5; the visual keys
// and values are fixed once prefilled):
//   fq[h*nv + j][k] = sum_e K[h][j][e] * Wq[h*dh + e][k]   ([H*nv][d]: scores = fq . norm(x))
//   fo[n][h*nv + j] = sum_e Wo[n][h*dh + e] * V[h][j][e]   ([d][H*nv]: out = fo . softmax(scores))
// xk / xv: [H][nv][dh] of kvdtype; wq [H*dh][d], wo [d][H*dh] of wdtype.
bool cross_fold_ok(int nv, int dh);
hipError_t launch_cross_fold(const void* xk, const void* xv, int kvdtype, const void* wq,
                             const void* wo, int wdtype, int H, int nv, int dh, int d, float* fq,
                             float* fo, hipStream_t s);

// The scores of the folded cross-attention taken from the layer's input and attention output
// instead of its post-attention residual (one-row steps): with F = fold_q diag(g) (g the
// cross-attention RMSNorm gain) and W_o the self-attention output matrix, fg[j] = [F[j] | (F W_o)[j]]
// ([HN][d + HD] float32), so fg . [x; o] = F (x + W_o o).  fold_q [HN][d] float32, wo [d][HD] in
// wdtype.
hipError_t launch_fold_fg(const float* fold_q, const float* gain, const void* wo, int wdtype,
                          int HN, int d, int HD, float* fg, hipStream_t s);

// Row statistics for normalisation: stats[m] = (mean, 1/sqrt(var+eps)) (LN) or (0, 1/rms) (RMS).
hipError_t launch_row_stats(const float* x, int ldx, int M, int K, int norm, float eps,
                            float2* stats, hipStream_t s);

// Confidence-stopped drafting, evaluated by the final argmax of draft step `step` (row m =
// sequence m): conf = the row's largest softmax probability, 1 / sum_n exp(logits[n] - max),
// from its logits (logits + m * ldl, V of them), stored at conf[m * ldc + step] when conf is set.
// Step 0 sets ndraft[m] = 1 and drafting[m] = (conf >= tau) for an active sequence (0 and 0 for
// an inactive one); a later step counts itself in ndraft[m] = step + 1 and updates drafting[m]
// only while drafting[m] is set.  logits == null: off.
struct ConfArgs {
  const float* logits = nullptr;
  int ldl = 0;
  int V = 0;
  float* conf = nullptr;
  int ldc = 0;
  int step = 0;
  float tau = 0.f;
  int32_t* drafting = nullptr;
  int32_t* ndraft = nullptr;
  const int32_t* active = nullptr;
};

// Final argmax over partials: tok = argmax; written to dst0[row_map(m)] and dst1[m] if set.
// Row m = b*C + j maps to dst0[b*ld0 + off0 + j].
hipError_t launch_argmax_final(const float* part_val, const int* part_idx, int M, int n_parts,
                               int C, int32_t* dst0, int ld0, int off0, int32_t* dst1,
                               hipStream_t s);
// The same, and the chosen token's embedding row (embed [vocab][d] in wdtype) into x_out row m.
hipError_t launch_argmax_final_embed(const float* part_val, const int* part_idx, int M,
                                     int n_parts, int C, int32_t* dst0, int ld0, int off0,
                                     int32_t* dst1, const void* embed, int wdtype, int d,
                                     float* x_out, hipStream_t s);

// The general form: the chosen token's embedding row into x_out when embed is set, and the
// confidence bookkeeping when cf.logits is set.
hipError_t launch_argmax_final_ex(const float* part_val, const int* part_idx, int M, int n_parts,
                                  int C, int32_t* dst0, int ld0, int off0, int32_t* dst1,
                                  const void* embed, int wdtype, int d, float* x_out,
                                  const ConfArgs& cf, hipStream_t s);

// Read-only stream of `bytes` (a multiple of 16) at buf, one 16 KB chunk per block of 256
// threads; out (4096 floats) is a sink that keeps the loads.
hipError_t launch_read_probe(const void* buf, size_t bytes, float* out, hipStream_t s);

// dst[b * ld_dst + j] = src[b * ld_src + j] for b < B, j < n (token rows).
hipError_t launch_copy_tokens(int32_t* dst, int ld_dst, const int32_t* src, int ld_src, int B,
                              int n, hipStream_t s);

// Cross-attention K or V at prefill: src [B*Nv][H*dh] float32 -> dst [B][H][Nv][dh] kvdtype.
hipError_t launch_scatter_cross(const float* src, void* dst, int B, int Nv, int H, int dh,
                                int kvdtype, hipStream_t s);

// Verify with reused layer-k states: x[b*(g+1)+j] = j < g ? stash[b*ld_stash_b + j*d] : x1[b*d].
hipError_t launch_assemble(float* x, const float* stash, int ld_stash_b, const float* x1, int B,
                           int g, int d, hipStream_t s);

hipError_t launch_set_seq_len(int32_t* seq_len, int B, int value, hipStream_t s);

// dst[r][0..cols) = src[r][0..cols) for r < rows (row strides ldd, lds floats).
hipError_t launch_copy_rows(float* dst, int ldd, const float* src, int lds, int rows, int cols,
                            hipStream_t s);

struct AcceptArgs {
  int B, gamma;
  const int32_t* draft;   // [B][gamma]
  const int32_t* target;  // [B][gamma+1]
  int32_t* pending;
  int32_t* out;           // [B][gamma+1] or null
  int32_t* accept_len;    // [B] or null
  const int32_t* active;  // [B] or null
  const int32_t* ndraft;  // [B] or null: drafts proposed by sequence b this round (<= gamma)
  int32_t* seq_len;
  int max_seq;
  int next_need;          // positions a following round needs beyond seq_len (0: none known)
  int32_t* status;
  // generation bookkeeping (null when called through ssd_accept)
  int32_t* tokens;        // [B][T]
  int32_t* count;         // [B] emitted so far
  int32_t* active_rw;     // [B] cleared when count reaches T
  int T;
  int64_t* stats;         // [3]: rounds (added by thread 0), accepted, drafted
  int32_t* n_active;      // [4]: sequences still active, shortest seq_len among them, the
                          // device status word, and the most tokens an active sequence still
                          // needs
};
hipError_t launch_accept(const AcceptArgs& a, hipStream_t s);

// Speculative sampling (sample.hip).
struct AcceptSampleArgs {
  int B = 0, gamma = 0, vocab = 0;
  const int32_t* draft = nullptr;          // [B][gamma]
  const float* draft_logits = nullptr;     // [B][gamma][vocab]
  const float* target_logits = nullptr;    // [B][gamma + 1][vocab]
  const float* u = nullptr;                // [B][gamma + 1]: acceptance tests, then the sample
  float inv_tau = 1.f;
  int32_t* pending = nullptr;
  int32_t* out = nullptr;                  // [B][gamma + 1] or null
  int32_t* accept_len = nullptr;           // [B] or null
  const int32_t* active = nullptr;         // [B] or null
  int32_t* seq_len = nullptr;
  int max_seq = 0;
  int32_t* status = nullptr;
};
hipError_t launch_accept_sample(const AcceptSampleArgs& a, hipStream_t s);

// Row m = b * C + j of logits (stride ldl): token sampled from softmax(row / tau) with uniform
// u[b * ldu + uoff + j], written to dst0[b * ld0 + off0 + j] and dst1[m] (if set).
hipError_t launch_sample_rows(const float* logits, int ldl, int M, int V, float tau,
                              const float* u, int ldu, int uoff, int C, int32_t* dst0, int ld0,
                              int off0, int32_t* dst1, hipStream_t s);

struct GenInitArgs {
  int B, T;
  const int32_t* pending;
  int32_t* tokens;
  int32_t* count;
  int32_t* active;
  int64_t* stats;
  int32_t* n_active;        // [4]: as AcceptArgs::n_active
  const int32_t* seq_len;
  int32_t* status;
};
hipError_t launch_gen_init(const GenInitArgs& a, hipStream_t s);

// T5 bias-by-distance table: table[h][n] = rel_bias[bucket[n]][h].
hipError_t launch_bias_table(const float* rel_bias, const int32_t* bucket, int H, int max_seq,
                             float* table, hipStream_t s);


}  // namespace ssd
