// Host side of libssd: argument checks, workspace layout, tables, and the launch sequences of
// prefill, draft, verify, accept and the whole decode loop (Algorithm 1).
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstring>
#include <map>
#include <mutex>
#include <new>
#include <tuple>
#include <vector>

#include "kernels.h"
#include "ssd.h"

using namespace ssd;

namespace {

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

constexpr int MAX_LAYERS = 256;  // decoder layers a context holds descriptors for

// T5 decoder relative-position bucket of a query-minus-key distance n >= 0: distances below
// half the buckets are exact, larger ones are binned logarithmically up to max_dist.
int t5_bucket(int n, int buckets, int max_dist) {
  const int exact = buckets / 2;
  if (n < exact) return n;
  const double f = std::log((double)n / exact) / std::log((double)max_dist / exact) * (buckets - exact);
  const int b = exact + (int)f;
  return b < buckets - 1 ? b : buckets - 1;
}

struct Layout {
  size_t x, x1, qkv, q, attn, ffn, inh, xi, stash, vis, part_val, part_idx, stats, bias_tab,
      p_x, p_attn, p_ffn, ssq, attn_part, fold_q, fold_o,
      bucket, rope_cos, rope_sin, status, cur_tok, g_pending, g_draft, g_target,
      g_count, g_active, g_nactive, g_stats, g_ndraft, g_drafting, g_draft_w, conf_lg, gplanes,
      fold_fg, kpart, total;
  int rows_max, head_rows, parts_max, ctx_max, plane_rows, attn_rows;
  int gplane_rows = 0, gplane_ld = 0;  // tile-path input planes (0 rows: none)
  int kpart_max = 0;                   // K-range partials of the tile path's residual projections
  bool fold = false;  // the folded cross-attention matrices are carved (fold_q, fold_o)
  bool fg = false;    // and the scores-from-the-layer-input matrices of layers 1..k (fold_fg)
};

int ctx_len_max(const ssd_dims& d) {
  return d.max_prompt + (d.arch == SSD_ARCH_LLAMA ? d.n_visual : 0);
}

// One-sequence T5 contexts fold the cross-attention into two float32 matrices per layer (the
// visual keys are fixed after prefill): one-row steps then take two weight-streaming launches for
// it instead of a query projection, an attention launch and an output projection.  Needs a
// softmax group the one-row kernel supports and scores that fit the query buffer.
bool fold_cross(const ssd_dims& d) {
  return d.arch == SSD_ARCH_T5 && d.max_batch == 1 && cross_fold_ok(d.n_visual, d.d_head) &&
         d.n_visual <= d.d_head && (size_t)d.n_heads * d.n_visual <= 6144 && d.d_model <= 6144;
}

// With the cross-attention folded, the one-row steps of layers 1..k (draft steps, the verify's
// last row, greedy steps) also take the folded scores from the layer's input and its attention
// output, fg . [x; o] = F (x + W_o o) with F = fold_q diag(g): the output projection and the scores
// then run in one launch, and the 1 / rms of the new residual is applied to the scores inside the
// softmax of the next launch.  Needs bf16 weights, HD <= 2048 and d <= 2048 (the two halves of
// the launch; the next launch reads the new residual row whole) and d_ff >= d (the row is kept
// in the FFN buffer until the FFN).
bool fold_fg_ok(const ssd_dims& d) {
  const int HD = d.n_heads * d.d_head;
  return fold_cross(d) && d.wdtype == SSD_BF16 && HD <= 2048 && d.d_model <= 2048 &&
         d.d_ff >= d.d_model && d.d_model % 8 == 0 && HD % 8 == 0;
}

// Workspace layout: the scratch a chain of launches writes (residual rows, projections, operand
// planes, argmax partials, the layer-k stash ...), the tables, the folded cross-attention and
// the loop state of ssd_generate, each slice 256-byte aligned.
bool make_layout(const ssd_dims& d, Layout& L, bool allow_fold = true) {
  const size_t B = d.max_batch, G = d.max_gamma, D = d.d_model, HD = (size_t)d.n_heads * d.d_head;
  L.ctx_max = ctx_len_max(d);
  size_t rows = B * (G + 1);
  rows = rows > B * L.ctx_max ? rows : B * L.ctx_max;
  if (d.arch == SSD_ARCH_T5 && rows < B * d.n_visual) rows = B * d.n_visual;
  L.rows_max = (int)rows;
  L.head_rows = (int)(B * (G + 1));
  L.parts_max = argmax_parts_max(d.vocab);
  // bf16 hi / lo operand planes of the skinny MFMA path (plane_rows rows each: the largest verify
  // chunk, rounded up to 16, at most 128) and its partial sums of squares
  {
    size_t pr = B * (G + 1);
    // (T5: the visual rows too, so the prefill's cross K/V projections take the skinny path)
    if (d.arch == SSD_ARCH_T5 && B * (size_t)d.n_visual <= 128 && B * (size_t)d.n_visual > pr)
      pr = B * (size_t)d.n_visual;
    pr = pr < 16 ? 16 : (pr > 128 ? 128 : (pr + 15) / 16 * 16);
    L.plane_rows = (int)pr;
  }
  // key-split partials of the long-context attention (up to 16 query rows per sequence)
  L.attn_rows = (int)(B * 16);
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off = align_up(off + bytes, 256); return o; };
  auto lane = [&](Layout& X, size_t R, size_t head_rows) {
    const size_t PRz = (size_t)L.plane_rows;
    X.x = take(R * D * 4);
    X.x1 = take((B * D + HD) * 4);  // room for a one-row attention output right after the row
    X.qkv = take(R * 3 * HD * 4);
    X.q = take(R * HD * 4);
    X.attn = take(R * HD * 4);
    X.ffn = take(R * (size_t)d.d_ff * 4);
    X.inh = take(B * (size_t)d.in_hidden * 4);
    X.xi = take(B * D * 4);
    X.stash = take(B * (G + 1) * D * 4);
    X.part_val = take(head_rows * L.parts_max * 4);
    X.part_idx = take(head_rows * L.parts_max * 4);
    X.stats = take(R * 8);
    X.p_x = take(2 * PRz * D * 2);
    X.p_attn = take(2 * PRz * HD * 2);
    X.p_ffn = take(2 * PRz * (size_t)d.d_ff * 2);
    X.ssq = take((size_t)2 * skinny_blocks((int)D) * PRz * 4);  // up to two partials per tile
    X.attn_part = take((size_t)L.attn_rows * d.n_heads * ATTN_SPLITS_MAX * (d.d_head + 2) * 4);
    X.cur_tok = take(B * 4);
  };
  lane(L, rows, (size_t)L.head_rows);
  // bf16 hi / lo planes of a context block's input rows for the tile GEMM (prefill)
  {
    int ld = (int)D;
    if ((int)HD > ld) ld = (int)HD;
    if (d.d_ff > ld) ld = d.d_ff;
    L.gplane_ld = (ld + 7) / 8 * 8;
    L.gplane_rows = (int)rows;
    L.gplanes = take((size_t)2 * rows * L.gplane_ld * 2);
    // contexts beyond the skinny capacity and one 128-row tile: room for four K-range partials
    L.kpart_max = (rows > (size_t)L.plane_rows && rows > 128) ? 4 : 0;
    L.kpart = take((size_t)L.kpart_max * rows * D * 4);
  }
  L.vis = take(d.arch == SSD_ARCH_T5 ? B * (size_t)d.n_visual * D * 4 : 0);
  {
    L.fold = allow_fold && fold_cross(d);
    const size_t fold = L.fold ? (size_t)d.n_layers * d.n_heads * d.n_visual * D * 4 : 0;
    L.fold_q = take(fold);
    L.fold_o = take(fold);
    L.fg = L.fold && fold_fg_ok(d);
    L.fold_fg = take(L.fg ? (size_t)d.draft_layers * d.n_heads * d.n_visual * (D + HD) * 4 : 0);
  }
  L.bias_tab = take(d.arch == SSD_ARCH_T5 ? (size_t)d.n_heads * d.max_seq * 4 : 0);
  L.bucket = take(d.arch == SSD_ARCH_T5 ? (size_t)d.max_seq * 4 : 0);
  L.rope_cos = take(d.arch == SSD_ARCH_LLAMA ? (size_t)d.max_seq * (d.d_head / 2) * 4 : 0);
  L.rope_sin = take(d.arch == SSD_ARCH_LLAMA ? (size_t)d.max_seq * (d.d_head / 2) * 4 : 0);
  L.status = take(4);
  L.g_pending = take(B * 4);
  L.g_draft = take(B * (G > 0 ? G : 1) * 4);
  L.g_target = take(B * (G + 1) * 4);
  L.g_count = take(B * 4);
  L.g_active = take(B * 4);
  L.g_nactive = take(16);
  L.g_stats = take(3 * 8);
  // confidence-stopped drafting: per-sequence draft counts and flags, the drafts at row stride
  // max_gamma, and a logits row per sequence for the confidence
  L.g_ndraft = take(B * 4);
  L.g_drafting = take(B * 4);
  L.g_draft_w = take(B * (G > 0 ? G : 1) * 4);
  L.conf_lg = take(B * (size_t)d.vocab * 4);
  L.total = off;
  return true;
}

bool dims_ok(const ssd_dims* d) {
  if (!d) return false;
  if (d->arch != SSD_ARCH_T5 && d->arch != SSD_ARCH_LLAMA) return false;
  if (d->n_layers < 1 || d->n_layers > MAX_LAYERS || d->d_model < 64 || d->d_model % 64)
    return false;
  if (d->n_heads < 1 || (d->d_head != 64 && d->d_head != 128)) return false;
  if (d->d_ff < 64 || d->d_ff % 64 || d->vocab < 2) return false;
  if (d->in_hidden < 64 || d->in_hidden % 64) return false;
  if (d->draft_layers < 1 || d->draft_layers > d->n_layers) return false;
  if (d->wdtype != SSD_F32 && d->wdtype != SSD_BF16) return false;
  if (d->kvdtype != SSD_F32 && d->kvdtype != SSD_BF16) return false;
  if (d->max_batch < 1 || d->max_batch > 256) return false;
  if (d->max_gamma < 0 || d->max_gamma > 32) return false;
  if (d->max_seq < 2 || d->max_seq > 1024) return false;  // attention keeps rows of scores in LDS
  if (d->max_prompt < 1 || d->page_size < 1 || d->max_pages < 1) return false;
  if ((long long)d->max_pages * d->page_size < d->max_seq) return false;
  if (ctx_len_max(*d) > d->max_seq) return false;
  if (!(d->norm_eps > 0.f) || !(d->ln_eps > 0.f)) return false;
  if (d->arch == SSD_ARCH_T5) {
    if (d->n_visual < 1 || d->rel_buckets < 2 || d->rel_max_dist <= d->rel_buckets / 2) return false;
  } else {
    if (d->n_visual < 0 || !(d->rope_theta > 0.f)) return false;
  }
  return true;
}

struct GraphKey {
  int kind, B, gamma, reuse;
  const void *p0, *p1, *p2, *p3;
  int i0 = 0, i1 = 0;
  const void *p4 = nullptr, *p5 = nullptr;
  bool operator<(const GraphKey& o) const {
    return std::tie(kind, B, gamma, reuse, p0, p1, p2, p3, i0, i1, p4, p5) <
           std::tie(o.kind, o.B, o.gamma, o.reuse, o.p0, o.p1, o.p2, o.p3, o.i0, o.i1, o.p4, o.p5);
  }
};

}  // namespace

struct ssd_ctx {
  ssd_dims d;
  ssd_weights w;
  ssd_layer_weights layers[MAX_LAYERS];
  ssd_kv kv;
  hipStream_t stream;
  char* ws;
  Layout L;
  int32_t* h_status = nullptr;  // pinned [4 + 256]: ssd_generate's read-back of the active counts,
                                // then the drafting flags of confidence-stopped drafting
  // the prefill's second stream (folded-scores products, created on first use, default priority)
  hipStream_t side = nullptr;
  hipEvent_t ev_fork = nullptr, ev_join = nullptr;
  bool is_static = false;       // made by ssd_create_static: workspace = the device's scratch
  int static_dev = -1;
  bool prefilled = false;
  bool fold_ready = false;  // fold_q / fold_o hold the prefilled sequence's cross-attention
  bool fg_ready = false;    // fold_fg too (layers 1..k)
  // reuse bookkeeping: the last ssd_draft's arguments
  bool draft_valid = false;
  int draft_B = 0, draft_gamma = 0;
  const int32_t* draft_pending = nullptr;
  const int32_t* draft_out = nullptr;
  bool use_graphs = true;
  std::map<GraphKey, hipGraphExec_t> graphs;
  // hidden-state export (ssd_set_hidden_export): imitation-network features and layer-k rows of
  // each draft step, final rows of each verify
  float* ex_phi = nullptr;
  float* ex_xk = nullptr;
  float* ex_xl = nullptr;
  // kernel timing (ssd_profile_enable)
  bool profiling = false;
  std::vector<hipEvent_t> ev_pool;
  size_t ev_used = 0;
  double prof_bytes = 0.0;
  int64_t prof_launches = 0;

  template <typename T> T* at(size_t off) { return reinterpret_cast<T*>(ws + off); }
  size_t kv_layer_elems() const {
    return (size_t)kv.n_pages * d.n_heads * d.page_size * d.d_head;
  }
  size_t xkv_layer_elems() const {
    return (size_t)d.max_batch * d.n_heads * d.n_visual * d.d_head;
  }
  size_t kv_elem() const { return d.kvdtype == SSD_BF16 ? 2 : 4; }
  size_t fold_layer_elems() const { return (size_t)d.n_heads * d.n_visual * d.d_model; }
  float* fg_layer(int l) {
    return reinterpret_cast<float*>(ws + L.fold_fg) +
           (size_t)l * d.n_heads * d.n_visual * (d.d_model + d.n_heads * d.d_head);
  }
};

#define HIP_TRY(expr)                          \
  do {                                         \
    if ((expr) != hipSuccess) return SSD_ERR_HIP; \
  } while (0)

namespace {

PagedKV paged(ssd_ctx* c, int l, int pos_off) {
  PagedKV p;
  p.k = (char*)c->kv.k_pool + (size_t)l * c->kv_layer_elems() * c->kv_elem();
  p.v = (char*)c->kv.v_pool + (size_t)l * c->kv_layer_elems() * c->kv_elem();
  p.page_table = c->kv.page_table;
  p.max_pages = c->d.max_pages;
  p.page_size = c->d.page_size;
  p.n_pages = c->kv.n_pages;
  p.seq_len = c->kv.seq_len;
  p.pos_off = pos_off;
  return p;
}

// launch_linear; when profiling, the launches of the profiled GEMV instantiation carry a pair of
// events bound to their own dispatch (kernel execution time, as a kernel trace reports it)
hipError_t run_linear(ssd_ctx* c, const LinearArgs& a, int* n_parts = nullptr) {
  if (!c->profiling) return launch_linear(a, c->stream, n_parts);
  while (c->ev_pool.size() < c->ev_used + 2) {
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess) return hipErrorOutOfMemory;
    c->ev_pool.push_back(e);
  }
  LaunchTiming t;
  t.start = c->ev_pool[c->ev_used];
  t.stop = c->ev_pool[c->ev_used + 1];
  t.K = c->d.d_model;  // the one-row launches over the d_model-wide matrices
  hipError_t err = launch_linear(a, c->stream, n_parts, &t);
  if (err != hipSuccess || !t.timed) return err;
  c->ev_used += 2;
  c->prof_bytes += linear_bytes(a);
  c->prof_launches += 1;
  return hipSuccess;
}

LinearArgs lin(ssd_ctx* c) {
  LinearArgs a;
  a.wdtype = c->d.wdtype;
  a.stats = c->at<float2>(c->L.stats);
  if (c->L.gplane_rows > 0) {
    a.gemm_planes = c->at<bf16_t>(c->L.gplanes);
    a.gemm_plane_rows = c->L.gplane_rows;
    a.gemm_plane_ld = c->L.gplane_ld;
    if (c->L.kpart_max > 0) {
      a.kpart = c->at<float>(c->L.kpart);
      a.kpart_max = c->L.kpart_max;
      a.kpart_ld = (int)c->d.d_model;
    }
  }
  a.eps = c->d.norm_eps;
  return a;
}

// Layers l0..l1-1 over rows r = b*C + j at positions seq_len[b] + pos_off + j.  When stash is set
// the residual after layer stash_layer is also written to stash[b * ld_stash + ...].
int run_layers(ssd_ctx* c, float* x, int B, int C, int pos_off, int l0, int l1, int stash_layer,
               float* stash, int ld_stash) {
  const ssd_dims& d = c->d;
  hipStream_t s = c->stream;
  const int R = B * C, D = d.d_model, HD = d.n_heads * d.d_head;
  const bool t5 = d.arch == SSD_ARCH_T5;
  // 2..16 rows in bf16: MFMA with operands written once as bf16 (the verify chunk)
  const int PR = c->L.plane_rows;
  const bool skinny = R <= PR && skinny_ok(R, D, d.wdtype) && skinny_ok(R, HD, d.wdtype) &&
                      skinny_ok(R, d.d_ff, d.wdtype);
  float* qkv = c->at<float>(c->L.qkv);
  float* q = c->at<float>(c->L.q);
  float* attn = c->at<float>(c->L.attn);
  float* ffn = c->at<float>(c->L.ffn);
  int32_t* status = c->at<int32_t>(c->L.status);
  // skinny operands: bf16 planes written once by each producer (p_x: gain * residual for the
  // RMS-normalised projections, with per-block sums of squares in ssq; p_attn, p_ffn)
  bf16_t* p_x = c->at<bf16_t>(c->L.p_x);
  bf16_t* p_attn = c->at<bf16_t>(c->L.p_attn);
  bf16_t* p_ffn = c->at<bf16_t>(c->L.p_ffn);
  float* ssq = c->at<float>(c->L.ssq);
  const int nssq_resid = skinny_ssq_parts(D, R);
  int nssq = 1;  // partials behind the current p_x
  // one linear layer: the skinny MFMA path for a verify chunk, else the vector / tile paths
  auto linear = [&](LinearArgs& a, const bf16_t* in, int in_ld) -> hipError_t {
    if (!skinny) return run_linear(c, a);
    a.in_planes = in;
    a.in_ld = in_ld;
    a.plane_rows = PR;
    if (a.norm == NORM_RMS) { a.in_ssq = ssq; a.in_nssq = nssq; }
    return launch_linear_skinny(a, s);
  };
  // a residual projection also leaves the planes of gain_next * x for the next projection
  auto resid_out = [&](LinearArgs& a, const float* gain_next) {
    if (!skinny || !gain_next) return;
    a.out_planes = p_x; a.out_ld = D; a.out_ssq = ssq; a.out_gain = gain_next;
  };
  if (skinny) HIP_TRY(launch_skinny_prep(x, D, R, D, c->layers[l0].attn_norm, p_x, D, PR, ssq, s));
  for (int l = l0; l < l1; ++l) {
    const ssd_layer_weights& lw = c->layers[l];
    // self-attention
    LinearArgs a = lin(c);
    a.x = x; a.ldx = D; a.M = R; a.K = D;
    a.norm = NORM_RMS; a.gain = lw.attn_norm;
    a.w[0] = lw.wq; a.w[1] = lw.wk; a.w[2] = lw.wv; a.n_mats = 3; a.n_per = HD;
    a.epi = EPI_QKV; a.y = q; a.ldy = HD;
    a.kv = paged(c, l, pos_off); a.C = C; a.n_heads = d.n_heads; a.d_head = d.d_head;
    a.kvdtype = d.kvdtype; a.max_seq = d.max_seq; a.status = status;
    a.rope_cos = t5 ? nullptr : c->at<float>(c->L.rope_cos);
    a.rope_sin = t5 ? nullptr : c->at<float>(c->L.rope_sin);
    if (skinny || linear_is_vector(a)) {
      // rotary and the KV store fused into the projection's epilogue
      HIP_TRY(linear(a, p_x, D));
    } else {
      a.epi = EPI_STORE; a.y = qkv; a.ldy = 3 * HD;
      HIP_TRY(run_linear(c, a));
      RopeScatterArgs rs;
      rs.qkv = qkv; rs.q_out = q; rs.B = B; rs.C = C; rs.H = d.n_heads; rs.dh = d.d_head;
      rs.kvdtype = d.kvdtype; rs.kv = a.kv;
      rs.rope_cos = a.rope_cos; rs.rope_sin = a.rope_sin;
      rs.max_seq = d.max_seq; rs.status = status;
      HIP_TRY(launch_rope_scatter(rs, s));
    }
    // one-row steps of layers 1..k with fold_fg: the attention output goes right after the
    // residual row, so that [x; o] is one input row of the folded-scores GEMV
    const bool fg = t5 && c->fg_ready && R == 1 && l < d.draft_layers;
    AttnArgs at;
    at.q = q; at.out = fg ? x + D : attn; at.out_planes = skinny ? p_attn : nullptr;
    at.plane_rows = PR;
    at.part = c->at<float>(c->L.attn_part); at.part_rows = c->L.attn_rows;
    at.B = B; at.C = C; at.H = d.n_heads; at.dh = d.d_head;
    at.kvdtype = d.kvdtype; at.cross = 0; at.kv = paged(c, l, pos_off);
    at.bias = t5 ? c->at<float>(c->L.bias_tab) : nullptr;
    at.max_seq = d.max_seq; at.xk = at.xv = nullptr; at.n_keys = 0;
    at.scale = t5 ? 1.0f : (float)(1.0 / std::sqrt((double)d.d_head));
    at.status = status;
    HIP_TRY(launch_attention(at, s));
    if (fg) {
      // y = x + W_o o into the FFN buffer and the unnormalised scores fg . [x; o] in one launch,
      // then x = y + fold_o . softmax(scores / rms(y)) per head
      const int HN = d.n_heads * d.n_visual;
      float* ybuf = ffn;
      LinearArgs wo = lin(c);
      wo.x = x + D; wo.ldx = HD; wo.M = 1; wo.K = HD;
      wo.w[0] = lw.wo; wo.n_per = D; wo.epi = EPI_BIAS_RESID; wo.resid = x; wo.ldr = D;
      wo.y = ybuf; wo.ldy = D;
      LinearArgs sc = lin(c);
      sc.x = x; sc.ldx = D + HD; sc.M = 1; sc.K = D + HD;
      sc.w[0] = c->fg_layer(l); sc.wdtype = SSD_F32; sc.n_per = HN; sc.epi = EPI_STORE;
      sc.y = q; sc.ldy = HD;
      HIP_TRY(launch_linear_pair(wo, sc, s));
      a = lin(c);
      a.x = q; a.ldx = HD; a.M = 1; a.K = HN;
      a.norm = NORM_SOFTMAX; a.group = d.n_visual; a.pre_row = ybuf; a.pre_len = D;
      a.w[0] = c->at<float>(c->L.fold_o) + (size_t)l * c->fold_layer_elems(); a.wdtype = SSD_F32;
      a.n_per = D; a.epi = EPI_BIAS_RESID; a.resid = ybuf; a.ldr = D; a.y = x; a.ldy = D;
      HIP_TRY(run_linear(c, a));
    } else {
    a = lin(c);
    a.x = attn; a.ldx = HD; a.M = R; a.K = HD;
    a.w[0] = lw.wo; a.n_per = D; a.epi = EPI_RESID; a.y = x; a.ldy = D;
    resid_out(a, t5 ? lw.xattn_norm : lw.ffn_norm);
    HIP_TRY(linear(a, p_attn, HD));
    nssq = nssq_resid;
    // cross-attention to the visual tokens
    if (t5 && c->fold_ready && R == 1) {
      // folded: scores = fold_q . rmsnorm(x), then x += fold_o . softmax(scores) per head
      const int HN = d.n_heads * d.n_visual;
      a = lin(c);
      a.x = x; a.ldx = D; a.M = R; a.K = D;
      a.norm = NORM_RMS; a.gain = lw.xattn_norm;
      a.w[0] = c->at<float>(c->L.fold_q) + (size_t)l * c->fold_layer_elems(); a.wdtype = SSD_F32;
      a.n_per = HN; a.epi = EPI_STORE; a.y = q; a.ldy = HD;
      HIP_TRY(run_linear(c, a));
      a = lin(c);
      a.x = q; a.ldx = HD; a.M = R; a.K = HN;
      a.norm = NORM_SOFTMAX; a.group = d.n_visual;
      a.w[0] = c->at<float>(c->L.fold_o) + (size_t)l * c->fold_layer_elems(); a.wdtype = SSD_F32;
      a.n_per = D; a.epi = EPI_RESID; a.y = x; a.ldy = D;
      HIP_TRY(run_linear(c, a));
    } else if (t5 && skinny && c->fold_ready &&
               skinny_fold_ok(D, d.n_heads * d.n_visual, d.n_visual, R)) {
      // folded, for a verify chunk on half tiles (float32 matrices split into bf16 hi / lo in the
      // kernel): scores = fold_q . rmsnorm(x) per row, then x += fold_o . softmax(scores) per head
      // with the softmax taken in the second launch's input loads
      const int HN = d.n_heads * d.n_visual;
      a = lin(c);
      a.x = x; a.ldx = D; a.M = R; a.K = D;
      a.norm = NORM_RMS; a.gain = lw.xattn_norm;
      a.w[0] = c->at<float>(c->L.fold_q) + (size_t)l * c->fold_layer_elems(); a.wdtype = SSD_F32;
      a.n_per = HN; a.epi = EPI_STORE; a.y = q; a.ldy = HD;
      a.in_planes = p_x; a.in_ld = D; a.plane_rows = PR; a.in_ssq = ssq; a.in_nssq = nssq;
      HIP_TRY(launch_linear_skinny_fold(a, s));
      a = lin(c);
      a.x = q; a.ldx = HD; a.M = R; a.K = HN;
      a.norm = NORM_SOFTMAX; a.group = d.n_visual;
      a.w[0] = c->at<float>(c->L.fold_o) + (size_t)l * c->fold_layer_elems(); a.wdtype = SSD_F32;
      a.n_per = D; a.epi = EPI_RESID; a.y = x; a.ldy = D;
      a.in_f32 = q; a.in_ld = HD; a.plane_rows = PR;
      resid_out(a, lw.ffn_norm);
      HIP_TRY(launch_linear_skinny_fold(a, s));
    } else if (t5) {
      a = lin(c);
      a.x = x; a.ldx = D; a.M = R; a.K = D;
      a.norm = NORM_RMS; a.gain = lw.xattn_norm;
      a.w[0] = lw.xq; a.n_per = HD; a.epi = EPI_STORE; a.y = q; a.ldy = HD;
      HIP_TRY(linear(a, p_x, D));
      AttnArgs xa = at;
      xa.cross = 1;
      xa.bias = nullptr;
      xa.scale = 1.0f;
      xa.xk = (char*)c->kv.xk + (size_t)l * c->xkv_layer_elems() * c->kv_elem();
      xa.xv = (char*)c->kv.xv + (size_t)l * c->xkv_layer_elems() * c->kv_elem();
      xa.n_keys = d.n_visual;
      HIP_TRY(launch_attention(xa, s));
      a = lin(c);
      a.x = attn; a.ldx = HD; a.M = R; a.K = HD;
      a.w[0] = lw.xo; a.n_per = D; a.epi = EPI_RESID; a.y = x; a.ldy = D;
      resid_out(a, lw.ffn_norm);
      HIP_TRY(linear(a, p_attn, HD));
    }
    }
    // feed-forward
    a = lin(c);
    a.x = x; a.ldx = D; a.M = R; a.K = D;
    a.norm = NORM_RMS; a.gain = lw.ffn_norm;
    a.w[0] = lw.w_gate; a.w[1] = lw.w_up; a.n_mats = 2; a.n_per = d.d_ff;
    a.epi = t5 ? EPI_GATED_GELU : EPI_GATED_SILU; a.y = ffn; a.ldy = d.d_ff;
    if (skinny) { a.y = nullptr; a.out_planes = p_ffn; a.out_ld = d.d_ff; }
    HIP_TRY(linear(a, p_x, D));
    a = lin(c);
    a.x = ffn; a.ldx = d.d_ff; a.M = R; a.K = d.d_ff;
    a.w[0] = lw.w_down; a.n_per = D; a.epi = EPI_RESID; a.y = x; a.ldy = D;
    if (stash && l == stash_layer) { a.stash = stash; a.lds = ld_stash; }
    resid_out(a, l + 1 < l1 ? c->layers[l + 1].attn_norm : nullptr);
    HIP_TRY(linear(a, p_ffn, d.d_ff));
  }
  return SSD_OK;
}

// g = final RMSNorm + LM head, argmax per row.  Rows m of x (stride ldx) map to dst0 as in
// launch_argmax_final.
// embed_out (argmax only): the chosen tokens' embedding rows [M][d_model], the next draft step's
// input, written by the final argmax.
int run_head(ssd_ctx* c, const float* x, int ldx, int M, int C, float* logits, int ldl,
             int32_t* dst0, int ld0, int off0, int32_t* dst1, const float* u = nullptr,
             int ldu = 0, int uoff = 0, float tau = 0.f, float* embed_out = nullptr,
             const ConfArgs* cf = nullptr) {
  const ssd_dims& d = c->d;
  LinearArgs a = lin(c);
  a.x = x; a.ldx = ldx; a.M = M; a.K = d.d_model;
  a.norm = NORM_RMS; a.gain = c->w.final_norm;
  a.w[0] = c->w.lm_head; a.n_per = d.vocab; a.epi = EPI_ARGMAX;
  a.part_val = c->at<float>(c->L.part_val);
  a.part_idx = c->at<int>(c->L.part_idx);
  a.logits = logits; a.ldl = ldl;
  int n_parts = 0;
  if (M <= c->L.plane_rows && skinny_ok(M, d.d_model, d.wdtype)) {
    bf16_t* p_x = c->at<bf16_t>(c->L.p_x);
    float* ssq = c->at<float>(c->L.ssq);
    const int PR = c->L.plane_rows;
    HIP_TRY(launch_skinny_prep(x, ldx, M, d.d_model, c->w.final_norm, p_x, d.d_model, PR, ssq,
                               c->stream));
    a.in_planes = p_x; a.in_ld = d.d_model; a.in_ssq = ssq; a.in_nssq = 1; a.plane_rows = PR;
    HIP_TRY(launch_linear_skinny(a, c->stream, &n_parts));
  } else {
    HIP_TRY(run_linear(c, a, &n_parts));
  }
  if (u) {
    // sampled tokens: inverse CDF of softmax(logits / tau) per row (the logits are written above)
    HIP_TRY(launch_sample_rows(logits, ldl, M, d.vocab, tau, u, ldu, uoff, C, dst0, ld0, off0,
                               dst1, c->stream));
    return SSD_OK;
  }
  if (embed_out || cf) {
    HIP_TRY(launch_argmax_final_ex(a.part_val, a.part_idx, M, n_parts, C, dst0, ld0, off0, dst1,
                                   c->w.embed, d.wdtype, d.d_model, embed_out,
                                   cf ? *cf : ConfArgs(), c->stream));
    return SSD_OK;
  }
  HIP_TRY(launch_argmax_final(a.part_val, a.part_idx, M, n_parts, C, dst0, ld0, off0, dst1,
                              c->stream));
  return SSD_OK;
}

// Imitation network on the layer-k rows xk [B][D]: LN -> FC1 + b1 -> GELU into inh, then
// FC2 + b2 (+ xk when residual) into xi.  `between` runs after FC1 (the hidden-state export).
template <typename F>
int run_imitation(ssd_ctx* c, const float* xk, int B, F between) {
  const ssd_dims& d = c->d;
  const int D = d.d_model;
  float* inh = c->at<float>(c->L.inh);
  LinearArgs a = lin(c);
  a.x = xk; a.ldx = D; a.M = B; a.K = D;
  a.norm = NORM_LN; a.gain = c->w.in_ln_w; a.shift = c->w.in_ln_b; a.eps = d.ln_eps;
  a.w[0] = c->w.in_w1; a.n_per = d.in_hidden; a.epi = EPI_BIAS_GELU; a.bias = c->w.in_b1;
  a.y = inh; a.ldy = d.in_hidden;
  HIP_TRY(run_linear(c, a));
  HIP_TRY(between());
  a = lin(c);
  a.x = inh; a.ldx = d.in_hidden; a.M = B; a.K = d.in_hidden;
  a.w[0] = c->w.in_w2; a.n_per = D; a.epi = EPI_BIAS_RESID; a.bias = c->w.in_b2;
  a.resid = d.in_residual ? xk : nullptr; a.ldr = D; a.y = c->at<float>(c->L.xi); a.ldy = D;
  HIP_TRY(run_linear(c, a));
  return SSD_OK;
}

// gamma draft steps from `pending`; step i runs at positions seq_len + i and leaves its layer-k
// rows in the stash.
int draft_launches(ssd_ctx* c, int B, int gamma, const int32_t* pending, int32_t* draft,
                   float* logits, const float* u = nullptr, float tau = 0.f) {
  const ssd_dims& d = c->d;
  const int D = d.d_model;
  float* x = c->at<float>(c->L.x);
  float* inh = c->at<float>(c->L.inh);
  float* xi = c->at<float>(c->L.xi);
  float* stash = c->at<float>(c->L.stash);
  int32_t* cur = c->at<int32_t>(c->L.cur_tok);
  const int ld_stash = (d.max_gamma + 1) * D;
  // greedy drafts: the final argmax of step i also writes step i + 1's embedding rows into x
  const bool fuse_embed = !u;
  for (int i = 0; i < gamma; ++i) {
    if (i == 0 || !fuse_embed) {
      EmbedArgs e;
      e.x = x; e.B = B; e.C = 1; e.d = D; e.embed = c->w.embed; e.vocab = d.vocab;
      e.wdtype = d.wdtype; e.t0 = nullptr; e.t1 = i == 0 ? pending : cur; e.ld1 = 1;
      e.visual = nullptr; e.n_visual = d.n_visual; e.n_prefix = 0;
      e.status = c->at<int32_t>(c->L.status);
      HIP_TRY(launch_embed(e, c->stream));
    }
    int rc = run_layers(c, x, B, 1, i, 0, d.draft_layers, d.draft_layers - 1,
                        stash + (size_t)i * D, ld_stash);
    if (rc) return rc;
    rc = run_imitation(c, x, B, [&]() -> hipError_t {
      if (!c->ex_phi) return hipSuccess;
      // export: the imitation network's hidden features of step i, [B][gamma][in_hidden]
      hipError_t err = launch_copy_rows(c->ex_phi + (size_t)i * d.in_hidden, gamma * d.in_hidden,
                                        inh, d.in_hidden, B, d.in_hidden, c->stream);
      if (err != hipSuccess) return err;
      return launch_copy_rows(c->ex_xk + (size_t)i * D, gamma * D, stash + (size_t)i * D, ld_stash,
                              B, D, c->stream);
    });
    if (rc) return rc;
    rc = run_head(c, xi, D, B, 1, logits ? logits + (size_t)i * d.vocab : nullptr,
                  gamma * d.vocab, draft, gamma, i, cur, u, gamma, i, tau,
                  fuse_embed && i + 1 < gamma ? x : nullptr);
    if (rc) return rc;
  }
  return SSD_OK;
}

// Draft step i of confidence-stopped drafting (B sequences): the token of step i - 1 (or
// `pending`) at positions seq_len + i through layers 1..k (stash row i), the imitation network
// and g, with the logits kept (the caller's [B][gamma][V] when given, else a workspace row per
// sequence) for the confidence; the final argmax writes the draft to dwork[b][i] (row stride
// gamma), updates ndraft / drafting, and gathers step i + 1's embedding rows.
int draft_conf_step(ssd_ctx* c, int B, int gamma, int i, float tau, const int32_t* pending,
                    const int32_t* active, int32_t* dwork, float* logits, float* conf) {
  const ssd_dims& d = c->d;
  const int D = d.d_model;
  float* x = c->at<float>(c->L.x);
  float* stash = c->at<float>(c->L.stash);
  int32_t* cur = c->at<int32_t>(c->L.cur_tok);
  const int ld_stash = (d.max_gamma + 1) * D;
  if (i == 0) {
    EmbedArgs e;
    e.x = x; e.B = B; e.C = 1; e.d = D; e.embed = c->w.embed; e.vocab = d.vocab;
    e.wdtype = d.wdtype; e.t0 = nullptr; e.t1 = pending; e.ld1 = 1;
    e.visual = nullptr; e.n_visual = d.n_visual; e.n_prefix = 0;
    e.status = c->at<int32_t>(c->L.status);
    HIP_TRY(launch_embed(e, c->stream));
  }
  int rc = run_layers(c, x, B, 1, i, 0, d.draft_layers, d.draft_layers - 1,
                      stash + (size_t)i * D, ld_stash);
  if (rc) return rc;
  rc = run_imitation(c, x, B, []() { return hipSuccess; });
  if (rc) return rc;
  ConfArgs cf;
  float* lg = logits ? logits + (size_t)i * d.vocab : c->at<float>(c->L.conf_lg);
  cf.logits = lg;
  cf.ldl = logits ? gamma * d.vocab : d.vocab;
  cf.V = d.vocab;
  cf.conf = conf;
  cf.ldc = gamma;
  cf.step = i;
  cf.tau = tau;
  cf.drafting = c->at<int32_t>(c->L.g_drafting);
  cf.ndraft = c->at<int32_t>(c->L.g_ndraft);
  cf.active = active;
  return run_head(c, c->at<float>(c->L.xi), D, B, 1, lg, cf.ldl, dwork, gamma, i, cur, nullptr, 0,
                  0, 0.f, i + 1 < gamma ? x : nullptr, &cf);
}

// Verify with the layer-k reuse, first part: layers 1..k for the last position only (into x1);
// the other positions' layer-k rows are the draft's.
int verify_last_row(ssd_ctx* c, int B, int gamma, const int32_t* draft) {
  const ssd_dims& d = c->d;
  float* x1 = c->at<float>(c->L.x1);
  EmbedArgs e;
  e.x = x1; e.B = B; e.C = 1; e.d = d.d_model; e.embed = c->w.embed; e.vocab = d.vocab;
  e.wdtype = d.wdtype; e.t0 = nullptr; e.t1 = draft + (gamma - 1); e.ld1 = gamma;
  e.visual = nullptr; e.n_visual = d.n_visual; e.n_prefix = 0;
  e.status = c->at<int32_t>(c->L.status);
  HIP_TRY(launch_embed(e, c->stream));
  return run_layers(c, x1, B, 1, gamma, 0, d.draft_layers, -1, nullptr, 0);
}

// Second part: the gamma + 1 rows (stash rows 0..gamma-1, then x1) through layers k+1..L, g and
// the argmax per row.
int verify_deep(ssd_ctx* c, int B, int gamma, const float* stash, int32_t* target, float* logits) {
  const ssd_dims& d = c->d;
  const int D = d.d_model, C = gamma + 1;
  float* x = c->at<float>(c->L.x);
  HIP_TRY(launch_assemble(x, stash, (d.max_gamma + 1) * D, c->at<float>(c->L.x1), B, gamma, D,
                          c->stream));
  int rc = run_layers(c, x, B, C, 0, d.draft_layers, d.n_layers, -1, nullptr, 0);
  if (rc) return rc;
  if (c->ex_xl) {
    // export: the final residual rows (before g's norm), [B][gamma + 1][d_model]
    HIP_TRY(launch_copy_rows(c->ex_xl, D, x, D, B * C, D, c->stream));
  }
  return run_head(c, x, D, B * C, C, logits, d.vocab, target, C, 0, nullptr);
}

int verify_launches(ssd_ctx* c, int B, int gamma, const int32_t* pending, const int32_t* draft,
                    int reuse, int32_t* target, float* logits) {
  const ssd_dims& d = c->d;
  const int D = d.d_model, C = gamma + 1;
  float* x = c->at<float>(c->L.x);
  if (reuse) {
    const int rc = verify_last_row(c, B, gamma, draft);
    if (rc) return rc;
    return verify_deep(c, B, gamma, c->at<float>(c->L.stash), target, logits);
  }
  EmbedArgs e;
  e.x = x; e.B = B; e.C = C; e.d = D; e.embed = c->w.embed; e.vocab = d.vocab;
  e.wdtype = d.wdtype; e.t0 = pending; e.t1 = draft; e.ld1 = gamma;
  e.visual = nullptr; e.n_visual = d.n_visual; e.n_prefix = 0;
  e.status = c->at<int32_t>(c->L.status);
  HIP_TRY(launch_embed(e, c->stream));
  const int rc = run_layers(c, x, B, C, 0, 0, d.n_layers, -1, nullptr, 0);
  if (rc) return rc;
  if (c->ex_xl) {
    HIP_TRY(launch_copy_rows(c->ex_xl, D, x, D, B * C, D, c->stream));
  }
  return run_head(c, x, D, B * C, C, logits, d.vocab, target, C, 0, nullptr);
}

// Run `fn` directly or through a cached HIP graph keyed by the call's shape and pointers.
template <typename F>
int launch_maybe_graph(ssd_ctx* c, const GraphKey& key, F fn) {
  if (!c->use_graphs || c->profiling) return fn();
  auto it = c->graphs.find(key);
  if (it == c->graphs.end()) {
    if (hipStreamBeginCapture(c->stream, hipStreamCaptureModeThreadLocal) != hipSuccess)
      return SSD_ERR_HIP;
    int rc = fn();
    hipGraph_t g = nullptr;
    hipError_t ec = hipStreamEndCapture(c->stream, &g);
    if (rc != SSD_OK) {
      if (g) (void)hipGraphDestroy(g);
      return rc;
    }
    if (ec != hipSuccess || !g) return SSD_ERR_HIP;
    hipGraphExec_t ex = nullptr;
    ec = hipGraphInstantiate(&ex, g, nullptr, nullptr, 0);
    (void)hipGraphDestroy(g);
    if (ec != hipSuccess) return SSD_ERR_HIP;
    it = c->graphs.emplace(key, ex).first;
  }
  HIP_TRY(hipGraphLaunch(it->second, c->stream));
  return SSD_OK;
}

// Up to gamma confidence-stopped draft steps; after each step but the last, the drafting flags
// are read back (unless tau <= 0, where no sequence stops) and the steps end once no active
// sequence drafts.  The drafts of the steps run go to d_draft[b][0..steps) (row stride steps).
// Returns the steps run in *steps.
int draft_confident(ssd_ctx* c, int B, int gamma, float tau, const int32_t* pending,
                    const int32_t* active, int32_t* d_draft, float* logits, float* conf,
                    int* steps) {
  int32_t* dwork = c->at<int32_t>(c->L.g_draft_w);
  int32_t* drafting = c->at<int32_t>(c->L.g_drafting);
  int tbits = 0;
  std::memcpy(&tbits, &tau, sizeof(tbits));
  int n = 0;
  for (int i = 0; i < gamma; ++i) {
    GraphKey key{8, B, gamma, i, pending, active, logits, conf};
    key.i0 = tbits;
    int rc = launch_maybe_graph(c, key, [&]() {
      return draft_conf_step(c, B, gamma, i, tau, pending, active, dwork, logits, conf);
    });
    if (rc) return rc;
    n = i + 1;
    if (i + 1 < gamma && tau > 0.f) {
      int32_t local[256];
      int32_t* h = c->h_status ? c->h_status + 4 : local;
      HIP_TRY(hipMemcpyAsync(h, drafting, (size_t)B * 4, hipMemcpyDeviceToHost, c->stream));
      HIP_TRY(hipStreamSynchronize(c->stream));
      bool any = false;
      for (int b = 0; b < B; ++b) any = any || h[b] != 0;
      if (!any) break;
    }
  }
  HIP_TRY(launch_copy_tokens(d_draft, n, dwork, gamma, B, n, c->stream));
  *steps = n;
  return SSD_OK;
}

}  // namespace

namespace {

int check_create_args(const ssd_dims* dims, const ssd_weights* w, const ssd_kv* kv) {
  if (!dims_ok(dims)) return SSD_ERR_SHAPE;
  const ssd_dims& d = *dims;
  const bool t5 = d.arch == SSD_ARCH_T5;
  if (!w->embed || !w->lm_head || !w->final_norm || !w->in_ln_w || !w->in_ln_b || !w->in_w1 ||
      !w->in_b1 || !w->in_w2 || !w->in_b2 || !w->layers)
    return SSD_ERR_ARG;
  if (t5 && !w->rel_bias) return SSD_ERR_ARG;
  for (int l = 0; l < d.n_layers; ++l) {
    const ssd_layer_weights& lw = w->layers[l];
    if (!lw.attn_norm || !lw.wq || !lw.wk || !lw.wv || !lw.wo || !lw.ffn_norm || !lw.w_gate ||
        !lw.w_up || !lw.w_down)
      return SSD_ERR_ARG;
    if (t5 && (!lw.xattn_norm || !lw.xq || !lw.xk || !lw.xv || !lw.xo)) return SSD_ERR_ARG;
  }
  if (!kv->k_pool || !kv->v_pool || !kv->page_table || !kv->seq_len || kv->n_pages < 1)
    return SSD_ERR_ARG;
  if (t5 && (!kv->xk || !kv->xv)) return SSD_ERR_ARG;
  return SSD_OK;
}

// Host-computed table of n values, value(i) for i < n, copied into device memory at dst through a
// small stack buffer, one synchronous chunk at a time (no host heap).
template <typename T, typename F>
int upload_table(T* dst, size_t n, F value, hipStream_t s) {
  constexpr size_t CHUNK = 1024;
  T buf[CHUNK];
  for (size_t i0 = 0; i0 < n; i0 += CHUNK) {
    const size_t m = n - i0 < CHUNK ? n - i0 : CHUNK;
    for (size_t i = 0; i < m; ++i) buf[i] = value(i0 + i);
    HIP_TRY(hipMemcpyAsync(dst + i0, buf, m * sizeof(T), hipMemcpyHostToDevice, s));
    HIP_TRY(hipStreamSynchronize(s));
  }
  return SSD_OK;
}

// Fill a context whose dimensions and descriptors were checked: copy them, point it at its
// workspace, build the relative-bias (T5) or rotary (LLaMA) tables and clear the status word.
int init_ctx(ssd_ctx* c, const ssd_dims& d, const ssd_weights* w, const ssd_kv* kv, char* ws,
             const Layout& L, void* stream) {
  c->d = d;
  c->w = *w;
  for (int l = 0; l < d.n_layers; ++l) c->layers[l] = w->layers[l];
  c->w.layers = c->layers;
  c->kv = *kv;
  c->stream = reinterpret_cast<hipStream_t>(stream);
  c->ws = ws;
  c->L = L;
  if (d.arch == SSD_ARCH_T5) {
    int rc = upload_table(c->at<int32_t>(L.bucket), (size_t)d.max_seq, [&](size_t n) {
      return (int32_t)t5_bucket((int)n, d.rel_buckets, d.rel_max_dist);
    }, c->stream);
    if (rc) return rc;
    HIP_TRY(launch_bias_table(w->rel_bias, c->at<int32_t>(L.bucket), d.n_heads, d.max_seq,
                              c->at<float>(L.bias_tab), c->stream));
  } else {
    const int half = d.d_head / 2;
    auto angle = [&](size_t e) {
      const size_t p = e / half, i = e % half;
      return (double)p * std::pow((double)d.rope_theta, -2.0 * (double)i / d.d_head);
    };
    const size_t n = (size_t)d.max_seq * half;
    int rc = upload_table(c->at<float>(L.rope_cos), n, [&](size_t e) { return (float)std::cos(angle(e)); },
                          c->stream);
    if (rc) return rc;
    rc = upload_table(c->at<float>(L.rope_sin), n, [&](size_t e) { return (float)std::sin(angle(e)); },
                      c->stream);
    if (rc) return rc;
  }
  HIP_TRY(hipMemsetAsync(c->at<int32_t>(L.status), 0, 4, c->stream));
  HIP_TRY(hipStreamSynchronize(c->stream));
  return SSD_OK;
}

// The workspace of contexts made by ssd_create_static: one fixed array per device, resident from
// the library's load until the process ends.  Host code never passes `scratch` itself to a
// kernel or a copy (on the host it only names the symbol); it uses the device address that
// hipGetSymbolAddress returns for the current device, looked up once per device.
constexpr int STATIC_MAX_DEVICES = 64;
std::mutex g_static_mu;
char* g_scratch_ptr[STATIC_MAX_DEVICES] = {};
bool g_static_live[STATIC_MAX_DEVICES] = {};
alignas(ssd_ctx) unsigned char g_static_ctx_mem[STATIC_MAX_DEVICES][sizeof(ssd_ctx)];

}  // namespace

__device__ __align__(256) unsigned char scratch[SSD_STATIC_SCRATCH_BYTES];

namespace {

// Device address of `scratch` on device dev (current), looked up on the device's first use.
int static_scratch(int dev, char** out) {
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
      (void)hipGetLastError();
      return SSD_ERR_HIP;
    }
    g_scratch_ptr[dev] = reinterpret_cast<char*>(p);
  }
  *out = g_scratch_ptr[dev];
  return SSD_OK;
}

}  // namespace

extern "C" {

size_t ssd_workspace_bytes(const ssd_dims* dims) {
  if (!dims_ok(dims)) return 0;
  Layout L;
  make_layout(*dims, L);
  return L.total;
}

int ssd_create(const ssd_dims* dims, const ssd_weights* w, const ssd_kv* kv, void* d_workspace,
               size_t workspace_bytes, void* stream, ssd_ctx** out) {
  if (!out) return SSD_ERR_ARG;
  *out = nullptr;
  if (!dims || !w || !kv || !d_workspace) return SSD_ERR_ARG;
  int rc = check_create_args(dims, w, kv);
  if (rc) return rc;
  Layout L;
  make_layout(*dims, L);
  if (workspace_bytes < L.total) return SSD_ERR_CAPACITY;
  if (((uintptr_t)d_workspace) % 256) return SSD_ERR_ARG;
  ssd_ctx* c = new (std::nothrow) ssd_ctx();
  if (!c) return SSD_ERR_ARG;
  rc = init_ctx(c, *dims, w, kv, reinterpret_cast<char*>(d_workspace), L, stream);
  // ssd_generate's per-batch read-back lands in pinned host memory (pageable if unavailable)
  if (rc == SSD_OK &&
      hipHostMalloc(reinterpret_cast<void**>(&c->h_status), 16 + 4 * 256, hipHostMallocDefault) != hipSuccess) {
    c->h_status = nullptr;
    (void)hipGetLastError();
  }
  if (rc != SSD_OK) {
    delete c;
    return rc;
  }
  *out = c;
  return SSD_OK;
}

int ssd_create_static(const ssd_dims* dims, const ssd_weights* w, const ssd_kv* kv, void* stream,
                      ssd_ctx** out) {
  if (!out) return SSD_ERR_ARG;
  *out = nullptr;
  if (!dims || !w || !kv) return SSD_ERR_ARG;
  int rc = check_create_args(dims, w, kv);
  if (rc) return rc;
  Layout L;
  make_layout(*dims, L, /*allow_fold=*/false);
  if (L.total > SSD_STATIC_SCRATCH_BYTES) return SSD_ERR_CAPACITY;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return SSD_ERR_HIP;
  if (dev >= STATIC_MAX_DEVICES) return SSD_ERR_SHAPE;
  std::lock_guard<std::mutex> lock(g_static_mu);
  if (g_static_live[dev]) return SSD_ERR_STATE;
  char* ws = nullptr;
  rc = static_scratch(dev, &ws);
  if (rc) return rc;
  ssd_ctx* c = new (g_static_ctx_mem[dev]) ssd_ctx();
  c->is_static = true;
  c->static_dev = dev;
  c->use_graphs = false;  // instantiating a graph allocates
  rc = init_ctx(c, *dims, w, kv, ws, L, stream);
  if (rc != SSD_OK) {
    c->~ssd_ctx();
    return rc;
  }
  g_static_live[dev] = true;
  *out = c;
  return SSD_OK;
}

int ssd_prefill(ssd_ctx* c, int B, int P, const int32_t* d_prompt, const void* d_visual,
                int32_t* d_pending, float* d_logits) {
  if (!c || !d_prompt || !d_pending) return SSD_ERR_ARG;
  const ssd_dims& d = c->d;
  const bool t5 = d.arch == SSD_ARCH_T5;
  if (B < 1 || B > d.max_batch || P < 1 || P > d.max_prompt) return SSD_ERR_SHAPE;
  if (d.n_visual > 0 && !d_visual) return SSD_ERR_ARG;
  const int Cx = P + (t5 ? 0 : d.n_visual);
  if (Cx > d.max_seq) return SSD_ERR_CAPACITY;
  const int D = d.d_model, HD = d.n_heads * d.d_head;
  hipStream_t s = c->stream;
  float* x = c->at<float>(c->L.x);
  int32_t* status = c->at<int32_t>(c->L.status);
  c->draft_valid = false;
  bool side_used = false;
  HIP_TRY(launch_set_seq_len(c->kv.seq_len, B, 0, s));
  if (t5) {
    // cross-attention K/V of every layer from z
    float* vis = c->at<float>(c->L.vis);
    EmbedArgs ev;
    ev.x = vis; ev.B = B; ev.C = d.n_visual; ev.d = D; ev.embed = c->w.embed; ev.vocab = d.vocab;
    ev.wdtype = d.wdtype; ev.t0 = nullptr; ev.t1 = nullptr; ev.ld1 = 0;
    ev.visual = d_visual; ev.n_visual = d.n_visual; ev.n_prefix = d.n_visual; ev.status = status;
    HIP_TRY(launch_embed(ev, s));
    float* tmp = c->at<float>(c->L.qkv);
    // the visual rows as skinny operand planes once for all 2L projections, when they fit
    const int MV = B * d.n_visual, PR = c->L.plane_rows;
    const bool sk = MV <= PR && skinny_ok(MV, D, d.wdtype) && skinny_ok(MV, HD, d.wdtype);
    bf16_t* p_x = c->at<bf16_t>(c->L.p_x);
    if (sk)
      HIP_TRY(launch_skinny_prep(vis, D, MV, D, nullptr, p_x, D, PR, c->at<float>(c->L.ssq), s));
    for (int l = 0; l < d.n_layers; ++l) {
      for (int which = 0; which < 2; ++which) {
        LinearArgs a = lin(c);
        a.x = vis; a.ldx = D; a.M = MV; a.K = D;
        a.w[0] = which ? c->layers[l].xv : c->layers[l].xk; a.n_per = HD;
        a.epi = EPI_STORE; a.y = tmp; a.ldy = HD;
        if (sk) {
          a.in_planes = p_x; a.in_ld = D; a.plane_rows = PR;
          HIP_TRY(launch_linear_skinny(a, s));
        } else {
          HIP_TRY(run_linear(c, a));
        }
        void* dst = (char*)(which ? c->kv.xv : c->kv.xk) + (size_t)l * c->xkv_layer_elems() * c->kv_elem();
        HIP_TRY(launch_scatter_cross(tmp, dst, B, d.n_visual, d.n_heads, d.d_head, d.kvdtype, s));
      }
    }
    // The folded cross-attention of every layer (and the folded-scores products of layers 1..k)
    // on a second stream, beside the prompt's pass through the decoder, which leaves most of the
    // device idle and does not read them (that pass runs the cross-attention unfolded); the
    // context's stream waits for them before the prefill ends.  (Forking per layer, as soon as
    // each layer's cross K/V exist, measured no faster.)
    if (c->L.fold) {
      if (!c->side) {
        if (hipStreamCreateWithFlags(&c->side, hipStreamNonBlocking) != hipSuccess) {
          c->side = nullptr;
          return SSD_ERR_HIP;
        }
        if (hipEventCreateWithFlags(&c->ev_fork, hipEventDisableTiming) != hipSuccess ||
            hipEventCreateWithFlags(&c->ev_join, hipEventDisableTiming) != hipSuccess)
          return SSD_ERR_HIP;
      }
      HIP_TRY(hipEventRecord(c->ev_fork, s));
      HIP_TRY(hipStreamWaitEvent(c->side, c->ev_fork, 0));
      for (int l = 0; l < d.n_layers; ++l) {
        const size_t off = (size_t)l * c->xkv_layer_elems() * c->kv_elem();
        float* fq = c->at<float>(c->L.fold_q) + (size_t)l * c->fold_layer_elems();
        HIP_TRY(launch_cross_fold((char*)c->kv.xk + off, (char*)c->kv.xv + off, d.kvdtype,
                                  c->layers[l].xq, c->layers[l].xo, d.wdtype, d.n_heads,
                                  d.n_visual, d.d_head, D, fq,
                                  c->at<float>(c->L.fold_o) + (size_t)l * c->fold_layer_elems(),
                                  c->side));
        if (c->L.fg && l < d.draft_layers)
          HIP_TRY(launch_fold_fg(fq, c->layers[l].xattn_norm, c->layers[l].wo, d.wdtype,
                                 d.n_heads * d.n_visual, D, HD, c->fg_layer(l), c->side));
      }
      HIP_TRY(hipEventRecord(c->ev_join, c->side));
      side_used = true;
    }
  }
  // the prompt's pass reads the cross K/V, never the folds (which are still being formed)
  c->fold_ready = false;
  c->fg_ready = false;
  EmbedArgs e;
  e.x = x; e.B = B; e.C = Cx; e.d = D; e.embed = c->w.embed; e.vocab = d.vocab; e.wdtype = d.wdtype;
  e.t0 = nullptr; e.t1 = d_prompt; e.ld1 = P; e.visual = d_visual; e.n_visual = d.n_visual;
  e.n_prefix = t5 ? 0 : d.n_visual; e.status = status;
  HIP_TRY(launch_embed(e, s));
  int rc = run_layers(c, x, B, Cx, 0, 0, d.n_layers, -1, nullptr, 0);
  if (rc) return rc;
  rc = run_head(c, x + (size_t)(Cx - 1) * D, Cx * D, B, 1, d_logits, d.vocab, d_pending, 1, 0,
                nullptr);
  if (rc) return rc;
  HIP_TRY(launch_set_seq_len(c->kv.seq_len, B, Cx, s));
  if (side_used) HIP_TRY(hipStreamWaitEvent(s, c->ev_join, 0));
  c->fold_ready = t5 && c->L.fold;
  c->fg_ready = t5 && c->L.fg;
  c->prefilled = true;
  return SSD_OK;
}

int ssd_draft(ssd_ctx* c, int B, int gamma, const int32_t* d_pending, int32_t* d_draft,
              float* d_draft_logits) {
  if (!c || !d_pending || !d_draft) return SSD_ERR_ARG;
  if (B < 1 || B > c->d.max_batch || gamma < 1 || gamma > c->d.max_gamma) return SSD_ERR_SHAPE;
  if (!c->prefilled) return SSD_ERR_STATE;
  GraphKey key{0, B, gamma, 0, d_pending, d_draft, d_draft_logits, nullptr};
  int rc = launch_maybe_graph(c, key, [&]() {
    return draft_launches(c, B, gamma, d_pending, d_draft, d_draft_logits);
  });
  if (rc) return rc;
  c->draft_valid = true;
  c->draft_B = B;
  c->draft_gamma = gamma;
  c->draft_pending = d_pending;
  c->draft_out = d_draft;
  return SSD_OK;
}

int ssd_draft_sample(ssd_ctx* c, int B, int gamma, const int32_t* d_pending, const float* d_u,
                     float temperature, int32_t* d_draft, float* d_draft_logits) {
  if (!c || !d_pending || !d_draft || !d_u || !d_draft_logits) return SSD_ERR_ARG;
  if (!(temperature > 0.f) || !std::isfinite(temperature)) return SSD_ERR_ARG;
  if (B < 1 || B > c->d.max_batch || gamma < 1 || gamma > c->d.max_gamma) return SSD_ERR_SHAPE;
  if (!c->prefilled) return SSD_ERR_STATE;
  int tbits = 0;
  std::memcpy(&tbits, &temperature, sizeof(tbits));
  GraphKey key{3, B, gamma, tbits, d_pending, d_draft, d_draft_logits, d_u};
  int rc = launch_maybe_graph(c, key, [&]() {
    return draft_launches(c, B, gamma, d_pending, d_draft, d_draft_logits, d_u, temperature);
  });
  if (rc) return rc;
  c->draft_valid = true;
  c->draft_B = B;
  c->draft_gamma = gamma;
  c->draft_pending = d_pending;
  c->draft_out = d_draft;
  return SSD_OK;
}

int ssd_accept_sample(ssd_ctx* c, int B, int gamma, const int32_t* d_draft,
                      const float* d_draft_logits, const float* d_target_logits, const float* d_u,
                      float temperature, int32_t* d_pending, int32_t* d_out,
                      int32_t* d_accept_len, const int32_t* d_active) {
  if (!c || !d_target_logits || !d_pending || !d_u ||
      (gamma > 0 && (!d_draft || !d_draft_logits)))
    return SSD_ERR_ARG;
  if (!(temperature > 0.f) || !std::isfinite(temperature)) return SSD_ERR_ARG;
  if (B < 1 || B > c->d.max_batch || gamma < 0 || gamma > c->d.max_gamma) return SSD_ERR_SHAPE;
  if (!c->prefilled) return SSD_ERR_STATE;
  AcceptSampleArgs a;
  a.B = B; a.gamma = gamma; a.vocab = c->d.vocab; a.draft = d_draft;
  a.draft_logits = d_draft_logits; a.target_logits = d_target_logits; a.u = d_u;
  a.inv_tau = 1.0f / temperature; a.pending = d_pending; a.out = d_out;
  a.accept_len = d_accept_len; a.active = d_active; a.seq_len = c->kv.seq_len;
  a.max_seq = c->d.max_seq; a.status = c->at<int32_t>(c->L.status);
  HIP_TRY(launch_accept_sample(a, c->stream));
  c->draft_valid = false;
  return SSD_OK;
}

int ssd_verify(ssd_ctx* c, int B, int gamma, const int32_t* d_pending, const int32_t* d_draft,
               int reuse_hidden, int32_t* d_target, float* d_logits) {
  if (!c || !d_pending || !d_target || (gamma > 0 && !d_draft)) return SSD_ERR_ARG;
  if (B < 1 || B > c->d.max_batch || gamma < 0 || gamma > c->d.max_gamma) return SSD_ERR_SHAPE;
  if (!c->prefilled) return SSD_ERR_STATE;
  const int reuse = (reuse_hidden && gamma > 0) ? 1 : 0;
  if (reuse && !(c->draft_valid && c->draft_B == B && c->draft_gamma == gamma &&
                 c->draft_pending == d_pending && c->draft_out == d_draft))
    return SSD_ERR_STATE;
  GraphKey key{1, B, gamma, reuse, d_pending, d_draft, d_target, d_logits};
  return launch_maybe_graph(c, key, [&]() {
    return verify_launches(c, B, gamma, d_pending, d_draft, reuse, d_target, d_logits);
  });
}

int ssd_accept(ssd_ctx* c, int B, int gamma, const int32_t* d_draft, const int32_t* d_target,
               int32_t* d_pending, int32_t* d_out, int32_t* d_accept_len, const int32_t* d_active) {
  if (!c || !d_target || !d_pending || (gamma > 0 && !d_draft)) return SSD_ERR_ARG;
  if (B < 1 || B > c->d.max_batch || gamma < 0 || gamma > c->d.max_gamma) return SSD_ERR_SHAPE;
  if (!c->prefilled) return SSD_ERR_STATE;
  AcceptArgs a;
  std::memset(&a, 0, sizeof(a));
  a.B = B; a.gamma = gamma; a.draft = d_draft; a.target = d_target; a.pending = d_pending;
  a.out = d_out; a.accept_len = d_accept_len; a.active = d_active; a.seq_len = c->kv.seq_len;
  // the caller decides whether another round follows: only a length past the cache is flagged
  a.max_seq = c->d.max_seq; a.next_need = 0;
  a.status = c->at<int32_t>(c->L.status);
  HIP_TRY(launch_accept(a, c->stream));
  c->draft_valid = false;
  return SSD_OK;
}

int ssd_draft_confident(ssd_ctx* c, int B, int gamma, float threshold, const int32_t* d_pending,
                        const int32_t* d_active, int32_t* d_draft, int32_t* d_ndraft,
                        float* d_conf, float* d_draft_logits, int* h_steps) {
  if (!c || !d_pending || !d_draft || !d_ndraft || !h_steps) return SSD_ERR_ARG;
  if (!std::isfinite(threshold)) return SSD_ERR_ARG;
  if (B < 1 || B > c->d.max_batch || gamma < 1 || gamma > c->d.max_gamma) return SSD_ERR_SHAPE;
  if (!c->prefilled) return SSD_ERR_STATE;
  c->draft_valid = false;
  int steps = 0;
  int rc = draft_confident(c, B, gamma, threshold, d_pending, d_active, d_draft, d_draft_logits,
                           d_conf, &steps);
  if (rc) return rc;
  HIP_TRY(hipMemcpyAsync(d_ndraft, c->at<int32_t>(c->L.g_ndraft), (size_t)B * 4,
                         hipMemcpyDeviceToDevice, c->stream));
  *h_steps = steps;
  c->draft_valid = true;
  c->draft_B = B;
  c->draft_gamma = steps;
  c->draft_pending = d_pending;
  c->draft_out = d_draft;
  return SSD_OK;
}

int ssd_accept_counts(ssd_ctx* c, int B, int gamma, const int32_t* d_draft,
                      const int32_t* d_ndraft, const int32_t* d_target, int32_t* d_pending,
                      int32_t* d_out, int32_t* d_accept_len, const int32_t* d_active) {
  if (!c || !d_target || !d_pending || !d_ndraft || (gamma > 0 && !d_draft)) return SSD_ERR_ARG;
  if (B < 1 || B > c->d.max_batch || gamma < 0 || gamma > c->d.max_gamma) return SSD_ERR_SHAPE;
  if (!c->prefilled) return SSD_ERR_STATE;
  AcceptArgs a;
  std::memset(&a, 0, sizeof(a));
  a.B = B; a.gamma = gamma; a.draft = d_draft; a.target = d_target; a.pending = d_pending;
  a.out = d_out; a.accept_len = d_accept_len; a.active = d_active; a.ndraft = d_ndraft;
  a.seq_len = c->kv.seq_len; a.max_seq = c->d.max_seq; a.next_need = 0;
  a.status = c->at<int32_t>(c->L.status);
  HIP_TRY(launch_accept(a, c->stream));
  c->draft_valid = false;
  return SSD_OK;
}

int ssd_generate_confident(ssd_ctx* c, int B, int P, const int32_t* d_prompt,
                           const void* d_visual, int T, int gamma, float threshold,
                           int reuse_hidden, int32_t* d_tokens, int64_t* h_stats) {
  if (!c || !d_tokens || T < 1 || !std::isfinite(threshold)) return SSD_ERR_ARG;
  if (gamma < 1 || gamma > c->d.max_gamma) return SSD_ERR_SHAPE;
  if (B < 1 || B > c->d.max_batch) return SSD_ERR_SHAPE;
  const int Cx = P + (c->d.arch == SSD_ARCH_T5 ? 0 : c->d.n_visual);
  if (Cx + T + c->d.max_gamma > c->d.max_seq) return SSD_ERR_CAPACITY;
  int32_t* pending = c->at<int32_t>(c->L.g_pending);
  int32_t* draft = c->at<int32_t>(c->L.g_draft);
  int32_t* target = c->at<int32_t>(c->L.g_target);
  int32_t* count = c->at<int32_t>(c->L.g_count);
  int32_t* active = c->at<int32_t>(c->L.g_active);
  int32_t* n_active = c->at<int32_t>(c->L.g_nactive);
  int64_t* stats = c->at<int64_t>(c->L.g_stats);
  int rc = ssd_prefill(c, B, P, d_prompt, d_visual, pending, nullptr);
  if (rc) return rc;
  GenInitArgs gi{B, T, pending, d_tokens, count, active, stats, n_active, c->kv.seq_len,
                 c->at<int32_t>(c->L.status)};
  HIP_TRY(launch_gen_init(gi, c->stream));
  AcceptArgs a;
  std::memset(&a, 0, sizeof(a));
  a.B = B; a.target = target; a.pending = pending; a.draft = draft;
  a.ndraft = c->at<int32_t>(c->L.g_ndraft);
  a.seq_len = c->kv.seq_len; a.max_seq = c->d.max_seq; a.next_need = gamma + 1;
  a.status = c->at<int32_t>(c->L.status);
  a.tokens = d_tokens; a.count = count; a.active_rw = active; a.T = T; a.stats = stats;
  a.n_active = n_active;
  int32_t h_active[4] = {0, 0, 0, 0};
  for (int round = 0; round < T; ++round) {
    int32_t* dst = c->h_status ? c->h_status : h_active;
    HIP_TRY(hipMemcpyAsync(dst, n_active, 16, hipMemcpyDeviceToHost, c->stream));
    HIP_TRY(hipStreamSynchronize(c->stream));
    if (dst != h_active) std::memcpy(h_active, dst, 16);
    if (h_active[2] != 0) return SSD_ERR_DEVICE;
    if (h_active[0] == 0) break;
    int steps = 0;
    rc = draft_confident(c, B, gamma, threshold, pending, active, draft, nullptr, nullptr, &steps);
    if (rc) return rc;
    c->draft_valid = true;
    c->draft_B = B;
    c->draft_gamma = steps;
    c->draft_pending = pending;
    c->draft_out = draft;
    rc = ssd_verify(c, B, steps, pending, draft, reuse_hidden, target, nullptr);
    if (rc) return rc;
    a.gamma = steps;
    HIP_TRY(launch_accept(a, c->stream));
    c->draft_valid = false;
  }
  {
    int32_t* dst = c->h_status ? c->h_status : h_active;
    HIP_TRY(hipMemcpyAsync(dst, n_active, 16, hipMemcpyDeviceToHost, c->stream));
    if (h_stats) HIP_TRY(hipMemcpyAsync(h_stats, stats, 24, hipMemcpyDeviceToHost, c->stream));
    HIP_TRY(hipStreamSynchronize(c->stream));
    if (dst != h_active) std::memcpy(h_active, dst, 16);
    if (h_active[2] != 0) return SSD_ERR_DEVICE;
  }
  return SSD_OK;
}

int ssd_dynamic_gamma(int t, int d0, int n_max) {
  const double sig = 1.0 / (1.0 + std::exp(-0.01 * ((double)t - 0.5 * (double)n_max)));
  return d0 + (int)std::floor(10.0 * sig);
}

int ssd_generate(ssd_ctx* c, int B, int P, const int32_t* d_prompt, const void* d_visual, int T,
                 int gamma, int mode, int reuse_hidden, int32_t* d_tokens, int64_t* h_stats) {
  if (!c || !d_tokens || T < 1) return SSD_ERR_ARG;
  if (mode != SSD_MODE_GREEDY && mode != SSD_MODE_SPECULATIVE &&
      mode != SSD_MODE_SPECULATIVE_DYNAMIC)
    return SSD_ERR_ARG;
  const bool dynamic = mode == SSD_MODE_SPECULATIVE_DYNAMIC;
  const int g_max = mode == SSD_MODE_GREEDY ? 0 : (dynamic ? gamma + 9 : gamma);
  if (mode != SSD_MODE_GREEDY && (gamma < 1 || g_max > c->d.max_gamma)) return SSD_ERR_SHAPE;
  if (B < 1 || B > c->d.max_batch) return SSD_ERR_SHAPE;
  const int Cx = P + (c->d.arch == SSD_ARCH_T5 ? 0 : c->d.n_visual);
  if (Cx + T + c->d.max_gamma > c->d.max_seq) return SSD_ERR_CAPACITY;
  int32_t* pending = c->at<int32_t>(c->L.g_pending);
  int32_t* draft = c->at<int32_t>(c->L.g_draft);
  int32_t* target = c->at<int32_t>(c->L.g_target);
  int32_t* count = c->at<int32_t>(c->L.g_count);
  int32_t* active = c->at<int32_t>(c->L.g_active);
  int32_t* n_active = c->at<int32_t>(c->L.g_nactive);
  int64_t* stats = c->at<int64_t>(c->L.g_stats);
  int rc = ssd_prefill(c, B, P, d_prompt, d_visual, pending, nullptr);
  if (rc) return rc;
  GenInitArgs gi{B, T, pending, d_tokens, count, active, stats, n_active, c->kv.seq_len,
                 c->at<int32_t>(c->L.status)};
  HIP_TRY(launch_gen_init(gi, c->stream));
  AcceptArgs a;
  std::memset(&a, 0, sizeof(a));
  a.B = B; a.draft = draft; a.target = target; a.pending = pending;
  a.seq_len = c->kv.seq_len; a.max_seq = c->d.max_seq; a.next_need = g_max + 1;
  a.status = c->at<int32_t>(c->L.status);
  a.tokens = d_tokens; a.count = count; a.active_rw = active; a.T = T; a.stats = stats;
  a.n_active = n_active;
  // the read-back lands in the context's pinned buffer (a direct copy), else on the stack
  int32_t h_active[4] = {0, 0, 0, 0};
  int round = 0;
  while (round < T) {
    int32_t* dst = c->h_status ? c->h_status : h_active;
    HIP_TRY(hipMemcpyAsync(dst, n_active, 16, hipMemcpyDeviceToHost, c->stream));
    HIP_TRY(hipStreamSynchronize(c->stream));
    if (dst != h_active) std::memcpy(h_active, dst, 16);
    // a device status bit (bad token id, position past the cache, unmapped page) ends the loop
    if (h_active[2] != 0) return SSD_ERR_DEVICE;
    if (h_active[0] == 0) break;
    const int g = mode == SSD_MODE_GREEDY ? 0
                  : (dynamic ? ssd_dynamic_gamma(h_active[1], gamma, c->d.max_seq) : gamma);
    if (g > c->d.max_gamma) return SSD_ERR_SHAPE;
    a.gamma = g;
    // a round emits at most g + 1 tokens per sequence, so with a fixed g the next
    // ceil(need / (g + 1)) rounds are all needed (need: the most tokens an active sequence still
    // lacks) and go out without a read-back in between; d(t) reads the lengths every round
    int k = dynamic ? 1 : (h_active[3] + g) / (g + 1);
    if (k < 1) k = 1;
    for (int r = 0; r < k && round < T; ++r, ++round) {
      if (g > 0) {
        rc = ssd_draft(c, B, g, pending, draft, nullptr);
        if (rc) return rc;
      }
      rc = ssd_verify(c, B, g, pending, draft, g > 0 ? reuse_hidden : 0, target, nullptr);
      if (rc) return rc;
      HIP_TRY(launch_accept(a, c->stream));
      c->draft_valid = false;
    }
  }
  // the status word of the last batch of rounds, read with the statistics
  {
    int32_t* dst = c->h_status ? c->h_status : h_active;
    HIP_TRY(hipMemcpyAsync(dst, n_active, 16, hipMemcpyDeviceToHost, c->stream));
    if (h_stats) HIP_TRY(hipMemcpyAsync(h_stats, stats, 24, hipMemcpyDeviceToHost, c->stream));
    HIP_TRY(hipStreamSynchronize(c->stream));
    if (dst != h_active) std::memcpy(h_active, dst, 16);
    if (h_active[2] != 0) return SSD_ERR_DEVICE;
  }
  return SSD_OK;
}

int ssd_set_graphs(ssd_ctx* c, int enable) {
  if (!c) return SSD_ERR_ARG;
  c->use_graphs = enable != 0;
  return SSD_OK;
}

int ssd_set_hidden_export(ssd_ctx* c, float* d_phi, float* d_xk, float* d_xl) {
  if (!c) return SSD_ERR_ARG;
  const bool on = d_phi || d_xk || d_xl;
  if (on && !(d_phi && d_xk && d_xl)) return SSD_ERR_ARG;
  if (c->ex_phi != d_phi || c->ex_xk != d_xk || c->ex_xl != d_xl) {
    // captured launch sequences differ with and without the export
    for (auto& kv : c->graphs) (void)hipGraphExecDestroy(kv.second);
    c->graphs.clear();
  }
  c->ex_phi = d_phi;
  c->ex_xk = d_xk;
  c->ex_xl = d_xl;
  return SSD_OK;
}

int ssd_profile_enable(ssd_ctx* c, int enable) {
  if (!c) return SSD_ERR_ARG;
  c->profiling = enable != 0;
  return SSD_OK;
}

int ssd_profile_read(ssd_ctx* c, int64_t* launches, double* seconds, double* bytes) {
  if (!c) return SSD_ERR_ARG;
  if (hipStreamSynchronize(c->stream) != hipSuccess) return SSD_ERR_HIP;
  double total_ms = 0.0;
  for (size_t i = 0; i + 1 < c->ev_used; i += 2) {
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, c->ev_pool[i], c->ev_pool[i + 1]) != hipSuccess) return SSD_ERR_HIP;
    total_ms += ms;
  }
  if (launches) *launches = c->prof_launches;
  if (seconds) *seconds = total_ms * 1e-3;
  if (bytes) *bytes = c->prof_bytes;
  c->ev_used = 0;
  c->prof_bytes = 0.0;
  c->prof_launches = 0;
  return SSD_OK;
}

int ssd_read_bandwidth(const void* d_buf, size_t bytes, float* d_out, int reps, void* stream,
                       double* gbps) {
  if (!d_buf || !d_out || !gbps || reps < 1 || bytes < 16 || bytes % 16) return SSD_ERR_ARG;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) {
    if (e0) (void)hipEventDestroy(e0);
    return SSD_ERR_HIP;
  }
  double best = 0.0;
  int rc = SSD_OK;
  for (int r = 0; r <= reps && rc == SSD_OK; ++r) {
    float ms = 0.f;
    if (hipEventRecord(e0, s) != hipSuccess ||
        launch_read_probe(d_buf, bytes, d_out, s) != hipSuccess ||
        hipEventRecord(e1, s) != hipSuccess || hipEventSynchronize(e1) != hipSuccess ||
        hipEventElapsedTime(&ms, e0, e1) != hipSuccess) {
      rc = SSD_ERR_HIP;
      break;
    }
    const double rate = (double)bytes / (ms * 1e-3) / 1e9;
    if (r > 0 && rate > best) best = rate;  // the first pass warms up
  }
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  *gbps = best;
  return rc;
}

int ssd_sync_status(ssd_ctx* c, int32_t* status) {
  if (!c) return SSD_ERR_ARG;
  int32_t v = 0;
  if (hipStreamSynchronize(c->stream) != hipSuccess) return SSD_ERR_HIP;
  if (hipMemcpy(&v, c->at<int32_t>(c->L.status), 4, hipMemcpyDeviceToHost) != hipSuccess)
    return SSD_ERR_HIP;
  if (status) *status = v;
  if (v != 0) {
    if (hipMemset(c->at<int32_t>(c->L.status), 0, 4) != hipSuccess) return SSD_ERR_HIP;
    return SSD_ERR_DEVICE;
  }
  return SSD_OK;
}

const char* ssd_status_string(int code) {
  switch (code) {
    case SSD_OK: return "ok";
    case SSD_ERR_ARG: return "invalid argument";
    case SSD_ERR_SHAPE: return "unsupported shape";
    case SSD_ERR_CAPACITY: return "capacity exceeded";
    case SSD_ERR_HIP: return "HIP runtime error";
    case SSD_ERR_STATE: return "call out of order";
    case SSD_ERR_DEVICE: return "device status error";
    default: return "unknown status";
  }
}

void ssd_destroy(ssd_ctx* c) {
  if (!c) return;
  (void)hipStreamSynchronize(c->stream);
  for (auto& kv : c->graphs) (void)hipGraphExecDestroy(kv.second);
  for (hipEvent_t e : c->ev_pool) (void)hipEventDestroy(e);
  if (c->h_status) (void)hipHostFree(c->h_status);
  if (c->side) {
    (void)hipStreamSynchronize(c->side);
    (void)hipStreamDestroy(c->side);
  }
  if (c->ev_fork) (void)hipEventDestroy(c->ev_fork);
  if (c->ev_join) (void)hipEventDestroy(c->ev_join);
  if (c->is_static) {
    std::lock_guard<std::mutex> lock(g_static_mu);
    const int dev = c->static_dev;
    c->~ssd_ctx();
    g_static_live[dev] = false;
    return;
  }
  delete c;
}

}  // extern "C"
