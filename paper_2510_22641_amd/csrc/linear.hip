// Linear layers y = epilogue(W . norm(x)) for the decoder, the imitation network and the LM head.
//
// Paths:
//  * gemv1_kernel — one input row (the batch-1 draft and greedy steps): a wave holds the whole
//    input row in registers and streams two weight rows with 16-byte loads; the norm statistics
//    are wave reductions (RMSNorm folded into the epilogue as 1/rms).  Bound: HBM bytes of W.
//  * gemv_kernel — weight streaming for 2..8 rows in float32 (or rows longer than a batch): the
//    input rows are staged in LDS with the gain applied, one row pair per wave.
//  * gemv_mfma_kernel — 2..128 rows with bf16 weights (the verify chunk, batch-8 draft steps):
//    16 features x 16 rows per block on v_mfma_f32_16x16x32_bf16, weights straight from HBM,
//    inputs as bf16 hi / lo planes written once by their producer.  Bound: HBM bytes of W.
//  * gemm_kernel — 64x64x64 tiles on v_mfma_f32_16x16x32_bf16 with LDS staging, for larger M
//    (prefill).  The fp32 inputs are normalised and split into bf16 hi / lo planes while staged.
//
// Every path accumulates in fp32 and ends in a fused epilogue (store, residual (+ stash), gated
// activation, bias + GELU, bias + residual, per-block (max, argmax) partials for the LM head, or
// QKV with rotary and the paged KV store).
#include "device.h"
#include "gemv_common.h"
#include "kernels.h"

#include <hip/hip_ext.h>

#include <climits>

namespace ssd {

namespace {

// Weight-streaming GEMV for MB <= 8 input rows held in LDS (MB * K <= GV_LDS_FLOATS).
// One row pair per wave (blockIdx.x * 4 + wave); a wave requests a whole batch (GV_KP * 512
// elements of both rows; the whole row for K <= 6144) at once and the many resident waves of a CU
// hide the memory latency.
// RMSNorm is folded: LDS holds gain * x and the per-row 1/rms multiplies the dot products in the
// epilogue; LayerNorm inputs are normalised while staged.
// (The wave index goes through readfirstlane in these kernels so that the compiler treats the
// wave's row choice as uniform: the matrix pointers then come from scalar registers instead of
// vector loads of the argument buffer that would wait for the inputs.)
template <typename WT, int MB, int GV_KP>
__global__ __launch_bounds__(256) void gemv_kernel(const LinearArgs a) {
  extern __shared__ float xs[];  // [MB][ldxs]
  __shared__ float red[GV_WAVES][2 * MB];
  __shared__ float rv[GV_WAVES][MB];
  __shared__ int ri[GV_WAVES][MB];

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int K = a.K;
  const int ldxs = (K + 7) & ~7;
  const int m0 = blockIdx.y * MB;
  const int mrows = min(MB, a.M - m0);
  const bool gated = (a.epi == EPI_GATED_GELU || a.epi == EPI_GATED_SILU);
  const bool argmax = a.epi == EPI_ARGMAX;
  const int n_total = gated ? a.n_per : a.n_per * a.n_mats;
  const int n_pairs = gated ? a.n_per : (n_total + 1) / 2;
  const int pr = blockIdx.x * GV_WAVES + wave;
  const bool rms = a.norm == NORM_RMS, ln = a.norm == NORM_LN;

  // inputs first: the wait counter is in order, so they must be requested before the weights
  float p2[MB];
#pragma unroll
  for (int m = 0; m < MB; ++m) p2[m] = 0.f;
  if (ln) {
    // LayerNorm: statistics first, then the normalised rows
    float p1[MB];
#pragma unroll
    for (int m = 0; m < MB; ++m) p1[m] = 0.f;
    for (int idx = tid * 4; idx < MB * ldxs; idx += 1024) {
      const int m = idx / ldxs, k = idx - m * ldxs;
      if (m < mrows && k < K) {
        const float4 v = *reinterpret_cast<const float4*>(a.x + (size_t)(m0 + m) * a.ldx + k);
#pragma unroll
        for (int mm = 0; mm < MB; ++mm)
          if (mm == m) {
            p1[mm] += (v.x + v.y) + (v.z + v.w);
            p2[mm] += (v.x * v.x + v.y * v.y) + (v.z * v.z + v.w * v.w);
          }
      }
    }
#pragma unroll
    for (int m = 0; m < MB; ++m) { p1[m] = wave_sum(p1[m]); p2[m] = wave_sum(p2[m]); }
    if (lane == 0) {
#pragma unroll
      for (int m = 0; m < MB; ++m) { red[wave][2 * m] = p1[m]; red[wave][2 * m + 1] = p2[m]; }
    }
    __syncthreads();
    for (int idx = tid * 4; idx < MB * ldxs; idx += 1024) {
      const int m = idx / ldxs, k = idx - m * ldxs;
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
      if (m < mrows && k < K) {
        const float s1 = (red[0][2 * m] + red[1][2 * m]) + (red[2][2 * m] + red[3][2 * m]);
        const float s2 = (red[0][2 * m + 1] + red[1][2 * m + 1]) + (red[2][2 * m + 1] + red[3][2 * m + 1]);
        const float mean = s1 / (float)K;
        const float rstd = 1.0f / sqrtf(fmaxf(s2 / (float)K - mean * mean, 0.f) + a.eps);
        v = *reinterpret_cast<const float4*>(a.x + (size_t)(m0 + m) * a.ldx + k);
        const float4 g = *reinterpret_cast<const float4*>(a.gain + k);
        const float4 b = *reinterpret_cast<const float4*>(a.shift + k);
        v.x = (v.x - mean) * rstd * g.x + b.x;
        v.y = (v.y - mean) * rstd * g.y + b.y;
        v.z = (v.z - mean) * rstd * g.z + b.z;
        v.w = (v.w - mean) * rstd * g.w + b.w;
      }
      *reinterpret_cast<float4*>(xs + m * ldxs + xs_off(k, ldxs)) = v;
    }
  } else {
    // 8 float4 per thread requested together (a loop with one load per trip would pay one
    // memory round trip per trip)
    constexpr int SB = 8;
    for (int base = tid * 4; base < MB * ldxs; base += 1024 * SB) {
      float4 v[SB], g[SB];
#pragma unroll
      for (int u = 0; u < SB; ++u) {
        const int idx = base + u * 1024;
        const int m = idx / ldxs, k = idx - m * ldxs;
        v[u] = g[u] = make_float4(0.f, 0.f, 0.f, 0.f);
        if (idx < MB * ldxs && m < mrows && k < K) {
          v[u] = *reinterpret_cast<const float4*>(a.x + (size_t)(m0 + m) * a.ldx + k);
          if (rms) g[u] = *reinterpret_cast<const float4*>(a.gain + k);
        }
      }
#pragma unroll
      for (int u = 0; u < SB; ++u) {
        const int idx = base + u * 1024;
        if (idx >= MB * ldxs) break;
        const int m = idx / ldxs, k = idx - m * ldxs;
        float4 x4 = v[u];
        if (rms) {
#pragma unroll
          for (int mm = 0; mm < MB; ++mm)
            if (mm == m) p2[mm] += (x4.x * x4.x + x4.y * x4.y) + (x4.z * x4.z + x4.w * x4.w);
          x4.x *= g[u].x; x4.y *= g[u].y; x4.z *= g[u].z; x4.w *= g[u].w;
        }
        *reinterpret_cast<float4*>(xs + m * ldxs + xs_off(k, ldxs)) = x4;
      }
    }
    if (rms) {
#pragma unroll
      for (int m = 0; m < MB; ++m) p2[m] = wave_sum(p2[m]);
      if (lane == 0) {
#pragma unroll
        for (int m = 0; m < MB; ++m) red[wave][2 * m + 1] = p2[m];
      }
    }
  }

  // the residual values this wave's epilogue adds (lane 0), then the first weights
  const RowPair<WT> r = row_pair<WT>(a, gated, n_total, pr < n_pairs ? pr : 0);
  const bool live = pr < n_pairs;
  float yold[2][MB];
  if (lane == 0 && live && (a.epi == EPI_RESID || a.epi == EPI_BIAS_RESID)) {
    const float* src = a.epi == EPI_RESID ? a.y : a.resid;
    const int ld = a.epi == EPI_RESID ? a.ldy : a.ldr;
#pragma unroll
    for (int m = 0; m < MB; ++m) {
      yold[0][m] = (src && r.ok0 && m < mrows) ? src[(size_t)(m0 + m) * ld + r.n0] : 0.f;
      yold[1][m] = (src && r.ok1 && m < mrows) ? src[(size_t)(m0 + m) * ld + r.n1] : 0.f;
    }
  }
  Vec8<WT> w[2][GV_KP];
  load_pieces<WT, GV_KP>(w, r, 0, K, lane);
  __syncthreads();

  float rscale[MB];  // per input row: 1/rms (RMSNorm folded into the epilogue) or 1
#pragma unroll
  for (int m = 0; m < MB; ++m) {
    rscale[m] = 1.f;
    if (rms) {
      const float s2 = (red[0][2 * m + 1] + red[1][2 * m + 1]) + (red[2][2 * m + 1] + red[3][2 * m + 1]);
      rscale[m] = 1.0f / sqrtf(s2 / (float)K + a.eps);
    }
  }

  float acc[2][MB];
#pragma unroll
  for (int s = 0; s < 2; ++s)
#pragma unroll
    for (int m = 0; m < MB; ++m) acc[s][m] = 0.f;
  for (int e0 = 0; e0 < K; e0 += 512 * GV_KP) {
    if (e0 > 0) load_pieces<WT, GV_KP>(w, r, e0, K, lane);
    fma_pieces<WT, MB, GV_KP>(w, xs, ldxs, e0, K, lane, acc);
  }
#pragma unroll
  for (int m = 0; m < MB; ++m) {
    acc[0][m] = wave_sum(acc[0][m]) * rscale[m];
    acc[1][m] = wave_sum(acc[1][m]) * rscale[m];
  }
  gemv_finish<WT, MB>(a, r, acc, yold, live, gated, argmax, m0, mrows, tid, lane, wave, rv, ri);
}

// One input row, K <= 512 * KP: the register path of the draft and greedy steps.  A wave's 64
// lanes hold the whole input row in registers (lane l owns elements p*512 + 8l .. +7 of every
// piece p), so the norm statistics are wave reductions and nothing is staged in LDS: each wave
// requests its inputs, then both weight rows, then the norm's gain (and shift), and computes the
// statistics while the weights are in flight.  NORM is the input transform (a template parameter
// so that rows without one keep no gain registers); NORM_SOFTMAX turns the row into per-group
// softmax probabilities (the folded cross-attention's second product).
template <typename WT, int KP, int NORM>
__global__ __launch_bounds__(256) void gemv1_kernel(const LinearArgs a) {
  __shared__ float rv[GV_WAVES][1];
  __shared__ int ri[GV_WAVES][1];
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int K = a.K;
  const bool gated = (a.epi == EPI_GATED_GELU || a.epi == EPI_GATED_SILU);
  const bool argmax = a.epi == EPI_ARGMAX;
  const int n_total = gated ? a.n_per : a.n_per * a.n_mats;
  const int n_pairs = gated ? a.n_per : (n_total + 1) / 2;
  const int pr = blockIdx.x * GV_WAVES + wave;
  constexpr bool rms = NORM == NORM_RMS, ln = NORM == NORM_LN;

  // inputs first (the wait counter retires loads in issue order); clamped, never conditional
  float xv[KP][8];
#pragma unroll
  for (int p = 0; p < KP; ++p) {
    const int e = min(p * 512 + lane * 8, K - 8);
    const float4 x0 = *reinterpret_cast<const float4*>(a.x + e);
    const float4 x1 = *reinterpret_cast<const float4*>(a.x + e + 4);
    xv[p][0] = x0.x; xv[p][1] = x0.y; xv[p][2] = x0.z; xv[p][3] = x0.w;
    xv[p][4] = x1.x; xv[p][5] = x1.y; xv[p][6] = x1.z; xv[p][7] = x1.w;
  }
  // NORM_SOFTMAX with a pre-scale row: that row (at most 2048 floats) is requested with the
  // inputs, before the weights, so that its reduction and the softmax overlap the weight stream
  constexpr int PRE = NORM == NORM_SOFTMAX ? 8 : 1;
  float4 prev[PRE];
  if (NORM == NORM_SOFTMAX && a.pre_row) {
#pragma unroll
    for (int u = 0; u < PRE; ++u) {
      const int e = min(lane * 4 + u * 256, a.pre_len - 4);
      prev[u] = *reinterpret_cast<const float4*>(a.pre_row + e);
    }
  }
  const RowPair<WT> r = row_pair<WT>(a, gated, n_total, pr < n_pairs ? pr : 0);
  const bool live = pr < n_pairs;
  const bool qkv = a.epi == EPI_QKV;
  const int qpos = qkv ? qkv_pos(a, 0) : 0;  // requested before the weights
  float yold[2][1] = {{0.f}, {0.f}};
  if (lane == 0 && live && (a.epi == EPI_RESID || a.epi == EPI_BIAS_RESID)) {
    const float* src = a.epi == EPI_RESID ? a.y : a.resid;
    yold[0][0] = (src && r.ok0) ? src[r.n0] : 0.f;
    yold[1][0] = (src && r.ok1) ? src[r.n1] : 0.f;
  }
  Vec8<WT> w[2][KP];
  load_pieces<WT, KP>(w, r, 0, K, lane);
  QkvPre pre = {};
  if (qkv) {
    const int HD = a.n_per, mat = r.n0 >= HD ? (r.n0 >= 2 * HD ? 2 : 1) : 0;
    pre = qkv_pre(a, mat, r.n0 - mat * HD, 0, qpos);
  }
  Vec8<float> gv[rms || ln ? KP : 1], sv[ln ? KP : 1];
  if (rms || ln) {
#pragma unroll
    for (int p = 0; p < KP; ++p) gv[p].load(a.gain + min(p * 512 + lane * 8, K - 8));
  }
  if (ln) {
#pragma unroll
    for (int p = 0; p < KP; ++p) sv[p].load(a.shift + min(p * 512 + lane * 8, K - 8));
  }

  if (NORM == NORM_SOFTMAX) {
    // softmax over groups of a.group inputs: a group is a.group / 8 consecutive lanes of a piece
    // (512 is a multiple of the group, so groups never straddle pieces, and K of whole groups)
    const int gl = a.group >> 3;
    if (a.pre_row) {
      // scale by 1 / rms of the row the scores came from (every wave reads that row in full;
      // clamped re-reads past pre_len count as zero)
      float s2 = 0.f;
#pragma unroll
      for (int u = 0; u < PRE; ++u)
        if (lane * 4 + u * 256 < a.pre_len)
          s2 += (prev[u].x * prev[u].x + prev[u].y * prev[u].y) +
                (prev[u].z * prev[u].z + prev[u].w * prev[u].w);
      s2 = wave_sum(s2);
      const float sc = 1.0f / sqrtf(s2 / (float)a.pre_len + a.eps);
#pragma unroll
      for (int p = 0; p < KP; ++p)
#pragma unroll
        for (int e = 0; e < 8; ++e) xv[p][e] *= sc;
    }
#pragma unroll
    for (int p = 0; p < KP; ++p) {
      float m = xv[p][0];
#pragma unroll
      for (int e = 1; e < 8; ++e) m = fmaxf(m, xv[p][e]);
      for (int o = 1; o < gl; o <<= 1) m = fmaxf(m, __shfl_xor(m, o, SSD_WAVE));
      float sum = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        xv[p][e] = expf(xv[p][e] - m);
        sum += xv[p][e];
      }
      for (int o = 1; o < gl; o <<= 1) sum += __shfl_xor(sum, o, SSD_WAVE);
      const float inv = 1.0f / sum;
#pragma unroll
      for (int e = 0; e < 8; ++e) xv[p][e] *= inv;
    }
  }
  // pieces past K (clamped re-reads) count as zero
#pragma unroll
  for (int p = 0; p < KP; ++p)
    if (p * 512 + lane * 8 >= K) {
#pragma unroll
      for (int e = 0; e < 8; ++e) xv[p][e] = 0.f;
    }
  float rscale = 1.f;
  if (rms) {
    float s2 = 0.f;
#pragma unroll
    for (int p = 0; p < KP; ++p)
#pragma unroll
      for (int e = 0; e < 8; ++e) s2 = fmaf(xv[p][e], xv[p][e], s2);
    s2 = wave_sum(s2);
    rscale = 1.0f / sqrtf(s2 / (float)K + a.eps);
#pragma unroll
    for (int p = 0; p < KP; ++p) {
      float g[8];
      gv[p].to_f32(g);
#pragma unroll
      for (int e = 0; e < 8; ++e) xv[p][e] *= g[e];
    }
  } else if (ln) {
    float s1 = 0.f;
#pragma unroll
    for (int p = 0; p < KP; ++p)
#pragma unroll
      for (int e = 0; e < 8; ++e) s1 += xv[p][e];
    const float mean = wave_sum(s1) / (float)K;
    float s2 = 0.f;
#pragma unroll
    for (int p = 0; p < KP; ++p)
      if (p * 512 + lane * 8 < K) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float c = xv[p][e] - mean;
          s2 = fmaf(c, c, s2);
        }
      }
    const float rstd = 1.0f / sqrtf(wave_sum(s2) / (float)K + a.eps);
#pragma unroll
    for (int p = 0; p < KP; ++p) {
      float g[8], b[8];
      gv[p].to_f32(g);
      sv[p].to_f32(b);
#pragma unroll
      for (int e = 0; e < 8; ++e) xv[p][e] = (xv[p][e] - mean) * rstd * g[e] + b[e];
    }
  }

  float acc[2][1] = {{0.f}, {0.f}};
#pragma unroll
  for (int p = 0; p < KP; ++p) {
    if (p * 512 + lane * 8 < K) {
      float w0[8], w1[8];
      w[0][p].to_f32(w0);
      w[1][p].to_f32(w1);
      float t0 = acc[0][0], t1 = acc[1][0];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        t0 = fmaf(w0[e], xv[p][e], t0);
        t1 = fmaf(w1[e], xv[p][e], t1);
      }
      acc[0][0] = t0;
      acc[1][0] = t1;
    }
  }
  acc[0][0] = wave_sum(acc[0][0]) * rscale;
  acc[1][0] = wave_sum(acc[1][0]) * rscale;
  gemv_finish<WT, 1>(a, r, acc, yold, live, gated, argmax, 0, 1, tid, lane, wave, rv, ri, pre,
                     qkv);
}

// One input row, 2048 <= K <= 2048 * KP (no LayerNorm): the K range is split
// over the block's four waves instead of its rows.  A block owns the four row pairs of gemv1
// (eight weight rows); wave w reads elements p * 2048 + 512 w + 8 lane .. +7 of the input, of the
// gain and of all eight rows, so that each wave requests a quarter of the input and gain bytes
// gemv1 does for the same weight bytes (those extra requests, not the weights, limit gemv1).  The
// eight partial dot products of a lane are reduced over the wave by halving exchanges (three
// swaps leave each group of eight lanes one row), then over the waves through LDS; RMSNorm is
// folded as in gemv1 with the sum of squares reduced the same way.  Wave w finishes row pair w
// with gemv1's epilogue.
template <typename WT, int KP, int NORM>
__device__ __forceinline__ void gemv1k_body(const LinearArgs& a, const int blk) {
  static_assert(NORM != NORM_LN, "LayerNorm rows take gemv1_kernel");
  __shared__ float part[GV_WAVES][9];
  __shared__ float rv[GV_WAVES][1];
  __shared__ int ri[GV_WAVES][1];
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int K = a.K;
  const bool gated = (a.epi == EPI_GATED_GELU || a.epi == EPI_GATED_SILU);
  const bool argmax = a.epi == EPI_ARGMAX;
  const int n_total = gated ? a.n_per : a.n_per * a.n_mats;
  const int n_pairs = gated ? a.n_per : (n_total + 1) / 2;
  constexpr bool rms = NORM == NORM_RMS;

  // inputs first (the wait counter retires loads in issue order); clamped, never conditional
  float xv[KP][8];
#pragma unroll
  for (int p = 0; p < KP; ++p) {
    const int e = min(p * 2048 + wave * 512 + lane * 8, K - 8);
    const float4 x0 = *reinterpret_cast<const float4*>(a.x + e);
    const float4 x1 = *reinterpret_cast<const float4*>(a.x + e + 4);
    xv[p][0] = x0.x; xv[p][1] = x0.y; xv[p][2] = x0.z; xv[p][3] = x0.w;
    xv[p][4] = x1.x; xv[p][5] = x1.y; xv[p][6] = x1.z; xv[p][7] = x1.w;
  }
  const int pr = blk * GV_WAVES + wave;
  const RowPair<WT> r = row_pair<WT>(a, gated, n_total, pr < n_pairs ? pr : 0);
  const bool live = pr < n_pairs;
  const bool qkv = a.epi == EPI_QKV;
  const int qpos = qkv ? qkv_pos(a, 0) : 0;  // requested before the weights
  float yold[2][1] = {{0.f}, {0.f}};
  if (lane == 0 && live && (a.epi == EPI_RESID || a.epi == EPI_BIAS_RESID)) {
    const float* src = a.epi == EPI_RESID ? a.y : a.resid;
    yold[0][0] = (src && r.ok0) ? src[r.n0] : 0.f;
    yold[1][0] = (src && r.ok1) ? src[r.n1] : 0.f;
  }
  Vec8<WT> w[GV_WAVES][2][KP];
#pragma unroll
  for (int q = 0; q < GV_WAVES; ++q) {
    const int pq = blk * GV_WAVES + q;
    const RowPair<WT> rq = row_pair<WT>(a, gated, n_total, pq < n_pairs ? pq : 0);
#pragma unroll
    for (int p = 0; p < KP; ++p) {
      const int e = min(p * 2048 + wave * 512 + lane * 8, K - 8);
      w[q][0][p].load(rq.w0 + e);
      w[q][1][p].load(rq.w1 + e);
    }
  }
  Vec8<float> gv[rms ? KP : 1];
  if (rms) {
#pragma unroll
    for (int p = 0; p < KP; ++p) gv[p].load(a.gain + min(p * 2048 + wave * 512 + lane * 8, K - 8));
  }
  QkvPre pre = {};
  if (qkv) {
    const int HD = a.n_per, mat = r.n0 >= HD ? (r.n0 >= 2 * HD ? 2 : 1) : 0;
    pre = qkv_pre(a, mat, r.n0 - mat * HD, 0, qpos);
  }

  // pieces past K (clamped re-reads) count as zero
#pragma unroll
  for (int p = 0; p < KP; ++p)
    if (p * 2048 + wave * 512 + lane * 8 >= K) {
#pragma unroll
      for (int e = 0; e < 8; ++e) xv[p][e] = 0.f;
    }
  float s2 = 0.f;
  if (rms) {
#pragma unroll
    for (int p = 0; p < KP; ++p)
#pragma unroll
      for (int e = 0; e < 8; ++e) s2 = fmaf(xv[p][e], xv[p][e], s2);
    s2 = wave_sum(s2);
#pragma unroll
    for (int p = 0; p < KP; ++p) {
      float g[8];
      gv[p].to_f32(g);
#pragma unroll
      for (int e = 0; e < 8; ++e) xv[p][e] *= g[e];
    }
  }

  // acc[2q + s]: row s of pair q
  float acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = 0.f;
#pragma unroll
  for (int q = 0; q < GV_WAVES; ++q)
#pragma unroll
    for (int p = 0; p < KP; ++p) {
      float w0[8], w1[8];
      w[q][0][p].to_f32(w0);
      w[q][1][p].to_f32(w1);
      float t0 = acc[2 * q], t1 = acc[2 * q + 1];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        t0 = fmaf(w0[e], xv[p][e], t0);
        t1 = fmaf(w1[e], xv[p][e], t1);
      }
      acc[2 * q] = t0;
      acc[2 * q + 1] = t1;
    }
  // halving exchanges: after the swaps over lane bits 5, 4, 3 lane l holds a partial of row
  // (l >> 3) & 7, summed over its group of eight lanes by the last three steps
  const bool b5 = lane & 32, b4 = lane & 16, b3 = lane & 8;
  float u[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float mine = b5 ? acc[i + 4] : acc[i], other = b5 ? acc[i] : acc[i + 4];
    u[i] = mine + __shfl_xor(other, 32, SSD_WAVE);
  }
  float t[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const float mine = b4 ? u[i + 2] : u[i], other = b4 ? u[i] : u[i + 2];
    t[i] = mine + __shfl_xor(other, 16, SSD_WAVE);
  }
  float sres = (b3 ? t[1] : t[0]) + __shfl_xor(b3 ? t[0] : t[1], 8, SSD_WAVE);
  sres += __shfl_xor(sres, 4, SSD_WAVE);
  sres += __shfl_xor(sres, 2, SSD_WAVE);
  sres += __shfl_xor(sres, 1, SSD_WAVE);
  if ((lane & 7) == 0) part[wave][lane >> 3] = sres;
  if (rms && lane == 0) part[wave][8] = s2;
  __syncthreads();
  float rscale = 1.f;
  if (rms) {
    const float tot = (part[0][8] + part[1][8]) + (part[2][8] + part[3][8]);
    rscale = 1.0f / sqrtf(tot / (float)K + a.eps);
  }
  float res[2][1];
  res[0][0] = ((part[0][2 * wave] + part[1][2 * wave]) + (part[2][2 * wave] + part[3][2 * wave])) * rscale;
  res[1][0] = ((part[0][2 * wave + 1] + part[1][2 * wave + 1]) + (part[2][2 * wave + 1] + part[3][2 * wave + 1])) * rscale;
  gemv_finish<WT, 1>(a, r, res, yold, live, gated, argmax, 0, 1, tid, lane, wave, rv, ri, pre,
                     qkv);
}

template <typename WT, int KP, int NORM>
__global__ __launch_bounds__(256) void gemv1k_kernel(const LinearArgs a) {
  gemv1k_body<WT, KP, NORM>(a, blockIdx.x);
}

// Two one-row GEMVs over the same inputs in one launch: blocks [0, na) run `a` (bf16 weights,
// K <= 2048 * KPA), the others `b` (float32 weights, K <= 2048 * KPB); no input transform.
template <int KPA, int KPB>
__global__ __launch_bounds__(256) void gemv1k_pair_kernel(const LinearArgs a, const LinearArgs b,
                                                          const int na) {
  const int blk = blockIdx.x;
  if (blk < na) gemv1k_body<bf16_t, KPA, NORM_NONE>(a, blk);
  else gemv1k_body<float, KPB, NORM_NONE>(b, blk - na);
}

// ---------------------------------------------------------------------------------------------
// Skinny MFMA path: 2..128 input rows (the verify chunk), bf16 weights, 16 rows per grid row.
// A block owns NT tiles of 16 output features (the A rows of v_mfma_f32_16x16x32_bf16) and its 4
// waves split K; the input rows are the B columns, and every activation fragment a wave loads
// feeds the MFMAs of all NT tiles.  One tile per block for the projections whose tiles do not
// outnumber the compute units (their grids need the parallelism), up to three for those that do,
// four for the many tiles of the LM head (the launcher below; measured at the FlanT5-xl verify
// shapes, 6 rows: W_o 7.0 us with one tile against 15.7 with four; LM head 39 against 35).  The inputs arrive as two bf16 planes
// hi = bf16(v), lo = bf16(v - hi) of v = g * x (g the RMSNorm gain, or 1), written once by their
// producer; multiplying both planes keeps the activations at about 16 mantissa bits while the
// weights are read once.  RMSNorm is folded: 1/rms of each row comes from partial sums of squares
// the producer left, and scales the outputs.  Per 64-element step a lane reads 32 contiguous
// bytes of one row of each tile and 32 bytes of each plane; all loads of a batch (inputs first,
// then weights) are issued before the first MFMA, and the 4 partial tiles are summed through LDS
// before the fused epilogue.  For EPI_QKV a tile's rows r and r + 8 are the rotary pair
// (i, i + dh/2) of one head, so rotary and the KV store are done here.  A residual epilogue also
// writes the next launch's planes (of out_gain * y_new) and per-tile partial sums of squares of
// y_new.
// PACK (at most 8 input rows): the B operand's 16 columns carry the hi plane of rows 0..7 in
// columns 0..7 and the lo plane in columns 8..15, so one activation load and one MFMA per 32
// elements cover both planes (half the loads and MFMAs of the two-plane form); the epilogue adds
// column t + 8 to column t.
constexpr int SKW = 4;  // waves per skinny block
constexpr int SSQ_MAX = 256;  // partial sums of squares a skinny consumer reads (d_model <= 4096)

// SK: 64-element steps per batch of loads (chosen by the launcher from the steps of a wave).
template <bool GATED, bool RMS, int NT, bool PACK, int SK>
__global__ __launch_bounds__(64 * SKW) void gemv_mfma_kernel(const LinearArgs a) {
  constexpr int NB = GATED ? 2 : 1;
  constexpr int NG = 4 * SKW;                                 // groups of 16 threads
  __shared__ float part[SKW][NB][NT][16][17];
  __shared__ float fin[NB][NT][16][17];
  __shared__ float best_v[16][17];
  __shared__ int best_i[16][17];
  __shared__ float rs[16];
  __shared__ float sq[4][16];
  __shared__ float ssq_red[4 * SKW][16];

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int K = a.K, M = a.M;
  const int n_out = GATED ? a.n_per : a.n_per * a.n_mats;
  const int tiles = (n_out + 15) / 16;
  const bool qkv = !GATED && a.epi == EPI_QKV;
  const int grp = blockIdx.x;
  const int steps = K / 64;
  const int s_beg = (steps * wave) / SKW, s_end = (steps * (wave + 1)) / SKW;
  const int half = a.d_head >> 1, per_head = qkv ? half / 8 : 1;

  // QKV tiles: matrix, head and 8-column group of the rotary pairs
  auto qkv_tile = [&](int vt, int& mat, int& c) {
    const int m = vt / (a.n_heads * per_head);
    const int rem = vt - m * a.n_heads * per_head;
    const int h = rem / per_head, jb = rem - h * per_head;
    mat = m;
    c = h * a.d_head + 8 * jb;
  };
  const int r16 = lane & 15;
  const bf16_t* wrow[NB][NT];
#pragma unroll
  for (int j = 0; j < NT; ++j) {
    const int vt = grp * NT + j;
    int row;
    if (qkv) {
      int m, c;
      qkv_tile(vt < tiles ? vt : 0, m, c);
      row = m * a.n_per + c + (r16 & 7) + (r16 >= 8 ? half : 0);
    } else {
      row = vt * 16 + r16;
    }
    const int rr = (vt < tiles && row < n_out) ? row : 0;
    if (GATED) {
      wrow[0][j] = reinterpret_cast<const bf16_t*>(a.w[0]) + (size_t)rr * K;
      wrow[NB - 1][j] = reinterpret_cast<const bf16_t*>(a.w[1]) + (size_t)rr * K;
    } else {
      int v = rr;
      const void* base = a.w[0];
      if (v >= a.n_per) { v -= a.n_per; base = a.w[1]; if (v >= a.n_per) { v -= a.n_per; base = a.w[2]; } }
      wrow[0][j] = reinterpret_cast<const bf16_t*>(base) + (size_t)v * K;
    }
  }
  const int kq = (lane >> 4) * 16;  // this lane's 16 elements within a step
  const int t0 = blockIdx.y * 16;   // this block's first input row
  // B column lane % 16: input row t0 + lane % 16, or (PACK) row lane % 8 of the hi (columns
  // 0..7) or lo (columns 8..15) plane
  const int tok = PACK ? (lane & 7) : t0 + (lane & 15);
  const bool tok_ok = tok < M;
  const int PR = a.plane_rows;
  const bf16_t* brow = a.in_planes + ((size_t)(PACK && (lane & 8) ? PR : 0) + (tok_ok ? tok : 0)) * a.in_ld;
  const bf16_t* brow_lo = brow + (size_t)PR * a.in_ld;

  // values the epilogue needs, requested before the main batch (the wait counter retires loads
  // in issue order): the producer's partial sums of squares (RMSNorm; thread: row t0 + tid % 16,
  // partials tid / 16 + NG i) and the old residual values of this thread's outputs
  float sv[RMS ? SSQ_MAX / NG : 1];
  if (RMS) {
#pragma unroll
    for (int i = 0; i < SSQ_MAX / NG; ++i) {
      const int p = (tid >> 4) + NG * i;
      sv[i] = a.in_ssq[(size_t)min(p, a.in_nssq - 1) * PR + t0 + (tid & 15)];
    }
  }
  float y_old[NT];
#pragma unroll
  for (int j = 0; j < NT; ++j) {
    y_old[j] = 0.f;
    if (a.epi == EPI_RESID) {
      const int ry = min(t0 + (tid & 15), M - 1);
      const int ny = min((grp * NT + j) * 16 + ((tid >> 4) & 15), n_out - 1);
      y_old[j] = a.y[(size_t)ry * a.ldy + ny];
    }
  }

  f32x4_t acc[NB][NT];
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int j = 0; j < NT; ++j) acc[b][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  for (int s0 = s_beg; s0 < s_end; s0 += SK) {
    uint4 wv[NB][NT][SK][2], bv[SK][2], bl[SK][2];
    // inputs first (L2-resident, they arrive early), then the weights in step order: the wait
    // counter retires loads in issue order, so step u waits only for its own weights
#pragma unroll
    for (int u = 0; u < SK; ++u) {
      const int k0 = min(s0 + u, s_end - 1) * 64 + kq;
      const uint4* bp = reinterpret_cast<const uint4*>(brow + k0);
      bv[u][0] = bp[0];
      bv[u][1] = bp[1];
      if (!PACK) {
        const uint4* bq = reinterpret_cast<const uint4*>(brow_lo + k0);
        bl[u][0] = bq[0];
        bl[u][1] = bq[1];
      }
    }
#pragma unroll
    for (int u = 0; u < SK; ++u) {
      const int k0 = min(s0 + u, s_end - 1) * 64 + kq;
#pragma unroll
      for (int j = 0; j < NT; ++j)
#pragma unroll
        for (int b = 0; b < NB; ++b) {
          const uint4* wp = reinterpret_cast<const uint4*>(wrow[b][j] + k0);
          wv[b][j][u][0] = wp[0];
          wv[b][j][u][1] = wp[1];
        }
    }
    __builtin_amdgcn_sched_barrier(0);  // keep the whole batch in flight before the first MFMA
#pragma unroll
    for (int u = 0; u < SK; ++u) {
      // a step past this wave's range re-read a clamped step, and a row past M re-read row 0:
      // zero operands instead of a branch (a branch would let the compiler sink the loads into it
      // and serialise the batch)
      const bool use = tok_ok && (s0 + u < s_end);
      const uint4 z = make_uint4(0, 0, 0, 0);
      const uint4 b0 = use ? bv[u][0] : z, b1 = use ? bv[u][1] : z;
      const uint4 c0 = (use && !PACK) ? bl[u][0] : z, c1 = (use && !PACK) ? bl[u][1] : z;
#pragma unroll
      for (int j = 0; j < NT; ++j)
#pragma unroll
        for (int b = 0; b < NB; ++b) {
          const bf16x8_t w0 = *reinterpret_cast<const bf16x8_t*>(&wv[b][j][u][0]);
          const bf16x8_t w1 = *reinterpret_cast<const bf16x8_t*>(&wv[b][j][u][1]);
          acc[b][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w0, *reinterpret_cast<const bf16x8_t*>(&b0), acc[b][j], 0, 0, 0);
          if (!PACK)
            acc[b][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w0, *reinterpret_cast<const bf16x8_t*>(&c0), acc[b][j], 0, 0, 0);
          acc[b][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w1, *reinterpret_cast<const bf16x8_t*>(&b1), acc[b][j], 0, 0, 0);
          if (!PACK)
            acc[b][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w1, *reinterpret_cast<const bf16x8_t*>(&c1), acc[b][j], 0, 0, 0);
        }
    }
  }
  float sp = 0.f;
  if (RMS) {
#pragma unroll
    for (int i = 0; i < SSQ_MAX / NG; ++i) sp += ((tid >> 4) + NG * i < a.in_nssq) ? sv[i] : 0.f;
  }
  // D[feature][token]: lane holds features 4 * (lane / 16) + e, token lane % 16
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int j = 0; j < NT; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) part[wave][b][j][4 * (lane >> 4) + e][lane & 15] = acc[b][j][e];
  if (RMS) ssq_red[tid >> 4][tid & 15] = sp;
  __syncthreads();

  // the block's tiles summed over its waves: thread (feature f, row t) of the first 256 threads
  static_assert(SKW >= 4, "the epilogue needs 256 threads");
  const int f = (tid >> 4) & 15, t = tid & 15, tg = t0 + t;
  const bool lead = tid < 256;
  float tsum[NB][NT];
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      float v = 0.f;
#pragma unroll
      for (int w = 0; w < SKW; ++w) v += part[w][b][j][f][t];
      tsum[b][j] = v;
    }
  if (lead) {
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int j = 0; j < NT; ++j) fin[b][j][f][t] = tsum[b][j];
  }
  // output (feature ff, input row tt) of tile j: with PACK the hi and lo columns added (only
  // tt < 8 is used then)
  auto out_at = [&](int b, int j, int ff, int tt) {
    return PACK ? fin[b][j][ff][tt] + fin[b][j][ff][(tt + 8) & 15] : fin[b][j][ff][tt];
  };
  if (RMS && tid < 16) {
    float s2 = 0.f;
#pragma unroll
    for (int g = 0; g < NG; ++g) s2 += ssq_red[g][tid];
    rs[tid] = 1.0f / sqrtf(s2 / (float)K + a.eps);
  }
  __syncthreads();

  const float rscale = RMS ? rs[t] : 1.f;
  for (int j = 0; j < NT; ++j) {
    const int vt = grp * NT + j;
    if (vt >= tiles) break;  // uniform over the block
    const int n = vt * 16 + f;
    const float v = out_at(0, j, f, t) * rscale;
    if (a.epi == EPI_ARGMAX) {
      const bool ok = lead && tg < M && n < n_out;
      if (lead) {
        best_v[t][f] = ok ? v : -INFINITY;
        best_i[t][f] = ok ? n : INT_MAX;
      }
      if (ok && a.logits) a.logits[(size_t)tg * a.ldl + n] = v;
      __syncthreads();
      if (tid < 16 && t0 + tid < M) {
        float bvv = -INFINITY;
        int bi = INT_MAX;
        for (int ff = 0; ff < 16; ++ff) argmax_merge(bvv, bi, best_v[tid][ff], best_i[tid][ff]);
        a.part_val[(size_t)(t0 + tid) * a.n_parts + vt] = bvv;
        a.part_idx[(size_t)(t0 + tid) * a.n_parts + vt] = bi;
      }
      __syncthreads();
      continue;
    }
    if (a.epi == EPI_RESID) {
      // y_new, the next planes and this tile's partial sums of squares (all threads take part in
      // the reduction; rows past M or features past n_out contribute zero)
      const bool ok = lead && tg < M && n < n_out;
      float y2 = 0.f;
      if (ok) {
        const float tt = y_old[j] + v;
        a.y[(size_t)tg * a.ldy + n] = tt;
        if (a.stash) a.stash[(size_t)tg * a.lds + n] = tt;
        if (a.out_planes) {
          const float gv = a.out_gain ? a.out_gain[n] * tt : tt;
          const uint32_t hi = f32_to_bf16(gv);
          a.out_planes[(size_t)tg * a.out_ld + n] = (bf16_t)hi;
          a.out_planes[(size_t)(PR + tg) * a.out_ld + n] = (bf16_t)f32_to_bf16(gv - bf16_to_f32(hi));
        }
        y2 = tt * tt;
      }
      if (a.out_ssq) {
        // threads with the same t: lanes t, t+16, t+32, t+48 of the first four waves
        y2 += __shfl_xor(y2, 16, SSD_WAVE);
        y2 += __shfl_xor(y2, 32, SSD_WAVE);
        if (lead && lane < 16) sq[wave][lane] = y2;
        __syncthreads();
        if (tid < 16) a.out_ssq[(size_t)vt * PR + t0 + tid] = (sq[0][tid] + sq[1][tid]) + (sq[2][tid] + sq[3][tid]);
        __syncthreads();
      }
      continue;
    }
    if (!lead || tg >= M) continue;
    if (qkv) {
      int m, c;
      qkv_tile(vt, m, c);
      if (f < 8) qkv_store_pair(a, m, c + f, tg, v, out_at(0, j, f + 8, t) * rscale);
      continue;
    }
    if (n >= n_out) continue;
    if (GATED) {
      const float act = apply_epi_act(a.epi, v, out_at(NB - 1, j, f, t) * rscale);
      if (a.y) a.y[(size_t)tg * a.ldy + n] = act;
      if (a.out_planes) {
        const uint32_t hi = f32_to_bf16(act);
        a.out_planes[(size_t)tg * a.out_ld + n] = (bf16_t)hi;
        a.out_planes[(size_t)(PR + tg) * a.out_ld + n] = (bf16_t)f32_to_bf16(act - bf16_to_f32(hi));
      }
      continue;
    }
    float* yp = a.y + (size_t)tg * a.ldy + n;
    switch (a.epi) {
      case EPI_STORE: *yp = v; break;
      case EPI_BIAS_GELU: *yp = gelu_tanh(v + a.bias[n]); break;
      case EPI_BIAS_RESID: *yp = (a.resid ? a.resid[(size_t)tg * a.ldr + n] : 0.f) + (v + a.bias[n]); break;
      default: break;
    }
  }
}

// Half tiles: the skinny path for at most 8 input rows when a compute unit would otherwise issue
// more loads (launch_skinny_as compares the forms).  A half tile is 8 of a tile's 16 features:
// feature f (0..7) of half s is tile row 4 s + (f & 3) + 8 (f >> 2), so a half tile holds four
// whole rotary pairs of a QKV tile (features f and f + 4).  The A operand holds a half tile's 8
// features twice, A row i being feature i & 7 over elements 0..31 (i < 8) or 32..63 (i >= 8) of a
// 64-element step, and the B operand's columns are the 8 input rows over the same two halves; lane
// l then reads the 16 bytes at element 32 ((l >> 3) & 1) + 8 (l >> 4) of row l & 7, so the eight
// lanes of a row cover its whole 128 bytes.  D[f][t] + D[f + 8][t + 8] is the step's dot product
// (the other two quadrants are cross terms and are dropped); the hi and lo planes take one load
// each and every weight load feeds two MFMAs.  A block takes NH half tiles (h = NH * block + i)
// whose weight loads share the block's input loads.  The epilogue runs on 64 threads per half tile
// (feature (tid / 8) % 8, row tid % 8); a residual epilogue leaves one partial sum of squares per
// half tile.
// MODE 1 and 2 take float32 weights (the folded cross-attention matrices of a verify chunk): a lane
// reads its 8 elements as 32 bytes and splits them into bf16 hi / lo, and a step takes the products
// hi.hi, hi.lo and lo.hi (about 16 mantissa bits on both sides).  MODE 2 also takes its input as
// float32 rows (in_f32) and turns them into softmax probabilities over groups of a.group
// consecutive inputs (8, 16 or 32: the group of a lane's 8 elements spans the 1, 2 or 4 lanes
// l, l ^ 16, l ^ 32, l ^ 48 of one row and step half), split into hi / lo as the B operand.
template <bool GATED, bool RMS, int NH, int SK, int MODE = 0>
__global__ __launch_bounds__(64 * SKW, 2) void gemv_mfma_half_kernel(const LinearArgs a) {
  constexpr int NB = GATED ? 2 : 1;
  constexpr int NG = 4 * SKW;  // groups of 16 threads
  constexpr bool WF = MODE >= 1, SMX = MODE == 2;
  static_assert(NH <= SKW, "one wave per half tile in the epilogue");
  static_assert(!WF || !GATED, "float32 weights: one matrix");
  __shared__ float part[SKW][NB][NH][8][9];
  __shared__ float rs[16];
  __shared__ float ssq_red[4 * SKW][16];

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int K = a.K, M = a.M;
  const int n_out = GATED ? a.n_per : a.n_per * a.n_mats;
  const int halves = 2 * ((n_out + 15) / 16);
  const bool qkv = !GATED && a.epi == EPI_QKV;
  const int steps = K / 64;
  const int s_beg = (steps * wave) / SKW, s_end = (steps * (wave + 1)) / SKW;
  const int dhalf = a.d_head >> 1, per_head = qkv ? dhalf / 8 : 1;
  const int h0 = blockIdx.x * NH;

  // QKV tiles: matrix, head and 8-column group of the rotary pairs
  auto qkv_tile = [&](int vt, int& mat, int& c) {
    const int m = vt / (a.n_heads * per_head);
    const int rem = vt - m * a.n_heads * per_head;
    const int hh = rem / per_head, jb = rem - hh * per_head;
    mat = m;
    c = hh * a.d_head + 8 * jb;
  };
  auto tile_row = [](int s, int f) { return 4 * s + (f & 3) + 8 * (f >> 2); };
  // output feature (or QKV weight row) of feature f of half tile h
  auto feature = [&](int h, int f) {
    const int vt = h >> 1, r16 = tile_row(h & 1, f);
    if (qkv) {
      int m, c;
      qkv_tile(vt, m, c);
      return m * a.n_per + c + (r16 & 7) + (r16 >= 8 ? dhalf : 0);
    }
    return vt * 16 + r16;
  };
  // this lane's weight rows: feature lane % 8 of each of the block's half tiles
  const bf16_t* wrow[NB][NH];
  const float* wrowf[NH];
#pragma unroll
  for (int i = 0; i < NH; ++i) {
    const int h = h0 + i;
    const int row = h < halves ? feature(h, lane & 7) : 0;
    const int rr = row < n_out ? row : 0;
    wrowf[i] = reinterpret_cast<const float*>(a.w[0]) + (size_t)rr * K;
    if (GATED) {
      wrow[0][i] = reinterpret_cast<const bf16_t*>(a.w[0]) + (size_t)rr * K;
      wrow[NB - 1][i] = reinterpret_cast<const bf16_t*>(a.w[1]) + (size_t)rr * K;
    } else {
      int v = rr;
      const void* base = a.w[0];
      if (v >= a.n_per) { v -= a.n_per; base = a.w[1]; if (v >= a.n_per) { v -= a.n_per; base = a.w[2]; } }
      wrow[0][i] = reinterpret_cast<const bf16_t*>(base) + (size_t)v * K;
    }
  }
  const int kq = ((lane >> 3) & 1) * 32 + (lane >> 4) * 8;  // this lane's 8 elements of a step
  const int tok = lane & 7;
  const bool tok_ok = tok < M;
  const int PR = a.plane_rows;
  const bf16_t* brow = a.in_planes + (size_t)(tok_ok ? tok : 0) * a.in_ld;
  const bf16_t* brow_lo = brow + (size_t)PR * a.in_ld;
  const float* frow = SMX ? a.in_f32 + (size_t)(tok_ok ? tok : 0) * a.in_ld : nullptr;
  const int gsh = SMX ? (a.group >= 32 ? 2 : (a.group >= 16 ? 1 : 0)) : 0;  // exchanges per group

  // epilogue thread: half tile ei, feature ef, row et
  const int ei = tid >> 6, ef = (tid >> 3) & 7, et = tid & 7;
  const int eh = h0 + ei;
  const bool elive = ei < NH && eh < halves;
  const int en = elive ? feature(eh, ef) : 0;

  // values the epilogue needs, requested before the main batch (the wait counter retires loads in
  // issue order): the producer's partial sums of squares (thread: row tid % 16, partials
  // tid / 16 + NG j) and the old residual value of this thread's output
  float sv[RMS ? SSQ_MAX / NG : 1];
  if (RMS) {
#pragma unroll
    for (int j = 0; j < SSQ_MAX / NG; ++j) {
      const int pp = (tid >> 4) + NG * j;
      sv[j] = a.in_ssq[(size_t)min(pp, a.in_nssq - 1) * PR + (tid & 15)];
    }
  }
  float y_old = 0.f;
  if (a.epi == EPI_RESID) y_old = a.y[(size_t)min(et, M - 1) * a.ldy + min(en, n_out - 1)];

  f32x4_t acc[NB][NH];
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int i = 0; i < NH; ++i) acc[b][i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  for (int s0 = s_beg; s0 < s_end; s0 += SK) {
    // bv: the hi and lo planes' 16 bytes (SMX: 32 bytes of the float32 row); wv: bf16 weights,
    // wf: float32 weights (WF)
    uint4 wv[NB][NH][WF ? 1 : SK], bv[SK][2];
    float4 wf[NH][WF ? SK : 1][2];
    // inputs first (L2-resident, they arrive early), then the weights in step order
#pragma unroll
    for (int u = 0; u < SK; ++u) {
      const int k0 = min(s0 + u, s_end - 1) * 64 + kq;
      if (SMX) {
        const float4 f0 = *reinterpret_cast<const float4*>(frow + k0);
        const float4 f1 = *reinterpret_cast<const float4*>(frow + k0 + 4);
        bv[u][0] = make_uint4(__float_as_uint(f0.x), __float_as_uint(f0.y), __float_as_uint(f0.z), __float_as_uint(f0.w));
        bv[u][1] = make_uint4(__float_as_uint(f1.x), __float_as_uint(f1.y), __float_as_uint(f1.z), __float_as_uint(f1.w));
      } else {
        bv[u][0] = *reinterpret_cast<const uint4*>(brow + k0);
        bv[u][1] = *reinterpret_cast<const uint4*>(brow_lo + k0);
      }
    }
#pragma unroll
    for (int u = 0; u < SK; ++u) {
      const int k0 = min(s0 + u, s_end - 1) * 64 + kq;
#pragma unroll
      for (int i = 0; i < NH; ++i) {
        if constexpr (WF) {
          wf[i][u][0] = *reinterpret_cast<const float4*>(wrowf[i] + k0);
          wf[i][u][1] = *reinterpret_cast<const float4*>(wrowf[i] + k0 + 4);
        } else {
#pragma unroll
          for (int b = 0; b < NB; ++b) wv[b][i][u] = *reinterpret_cast<const uint4*>(wrow[b][i] + k0);
        }
      }
    }
    __builtin_amdgcn_sched_barrier(0);  // keep the whole batch in flight before the first MFMA
#pragma unroll
    for (int u = 0; u < SK; ++u) {
      // a step past this wave's range, or a row past M, re-read valid data: zero operands
      const bool use = tok_ok && (s0 + u < s_end);
      const uint4 z = make_uint4(0, 0, 0, 0);
      uint4 b0 = bv[u][0], b1 = bv[u][1];
      if constexpr (SMX) {
        // softmax over the lane's group: max and sum over its 8 elements and the group's other
        // lanes (every lane takes part in the exchanges), then hi / lo of the probabilities
        float f[8] = {__uint_as_float(b0.x), __uint_as_float(b0.y), __uint_as_float(b0.z), __uint_as_float(b0.w),
                      __uint_as_float(b1.x), __uint_as_float(b1.y), __uint_as_float(b1.z), __uint_as_float(b1.w)};
        float m = f[0];
#pragma unroll
        for (int e = 1; e < 8; ++e) m = fmaxf(m, f[e]);
        const float m16 = fmaxf(m, __shfl_xor(m, 16, SSD_WAVE));
        const float m32 = fmaxf(m16, __shfl_xor(m16, 32, SSD_WAVE));
        m = gsh == 0 ? m : (gsh == 1 ? m16 : m32);
        float sum = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          f[e] = expf(f[e] - m);
          sum += f[e];
        }
        const float s16 = sum + __shfl_xor(sum, 16, SSD_WAVE);
        const float s32 = s16 + __shfl_xor(s16, 32, SSD_WAVE);
        sum = gsh == 0 ? sum : (gsh == 1 ? s16 : s32);
        const float inv = 1.0f / sum;
        split_bf16x8_v(make_float4(f[0] * inv, f[1] * inv, f[2] * inv, f[3] * inv),
                       make_float4(f[4] * inv, f[5] * inv, f[6] * inv, f[7] * inv), b0, b1);
      }
      // operands as values (no address taken, so that nothing of the batch lives in memory)
      const bf16x8_t B0 = __builtin_bit_cast(bf16x8_t, use ? b0 : z);
      const bf16x8_t B1 = __builtin_bit_cast(bf16x8_t, use ? b1 : z);
      if constexpr (WF) {
        // float32 weights: hi.hi, hi.lo and lo.hi
#pragma unroll
        for (int i = 0; i < NH; ++i) {
          uint4 whi, wlo;
          split_bf16x8_v(wf[i][u][0], wf[i][u][1], whi, wlo);
          const bf16x8_t Ah = __builtin_bit_cast(bf16x8_t, whi);
          const bf16x8_t Al = __builtin_bit_cast(bf16x8_t, wlo);
          acc[0][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Ah, B0, acc[0][i], 0, 0, 0);
          acc[0][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Ah, B1, acc[0][i], 0, 0, 0);
          acc[0][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Al, B0, acc[0][i], 0, 0, 0);
        }
      } else {
        // every weight fragment against the hi plane, then against the lo plane (independent
        // products back to back)
#pragma unroll
        for (int pl = 0; pl < 2; ++pl) {
#pragma unroll
          for (int i = 0; i < NH; ++i)
#pragma unroll
            for (int b = 0; b < NB; ++b)
              acc[b][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                  __builtin_bit_cast(bf16x8_t, wv[b][i][u]), pl ? B1 : B0, acc[b][i], 0, 0, 0);
        }
      }
    }
  }
  float sp = 0.f;
  if (RMS) {
#pragma unroll
    for (int j = 0; j < SSQ_MAX / NG; ++j) sp += ((tid >> 4) + NG * j < a.in_nssq) ? sv[j] : 0.f;
  }
  // lane holds D rows 4 (lane / 16) + e, column lane % 16: the useful quadrants are rows 0..7 x
  // columns 0..7 (lanes 0..7 and 16..23) and rows 8..15 x columns 8..15 (those lanes + 40)
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int i = 0; i < NH; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float v = acc[b][i][e] + __shfl_down(acc[b][i][e], 40, SSD_WAVE);
        if (lane < 24 && !(lane & 8)) part[wave][b][i][4 * (lane >> 4) + e][lane & 7] = v;
      }
  if (RMS) ssq_red[tid >> 4][tid & 15] = sp;
  __syncthreads();
  if (RMS && tid < 16) {
    float s2 = 0.f;
#pragma unroll
    for (int g = 0; g < NG; ++g) s2 += ssq_red[g][tid];
    rs[tid] = 1.0f / sqrtf(s2 / (float)K + a.eps);
  }
  __syncthreads();

  if (ei >= NH) return;  // whole waves
  const float rscale = RMS ? rs[et] : 1.f;
  auto sum_at = [&](int b, int f) {
    float v = 0.f;
#pragma unroll
    for (int w = 0; w < SKW; ++w) v += part[w][b][ei][f][et];
    return v * rscale;
  };
  const float v0 = sum_at(0, ef);
  const bool ok = elive && et < M && en < n_out;
  if (a.epi == EPI_RESID) {
    float y2 = 0.f;
    if (ok) {
      const float tt = y_old + v0;
      a.y[(size_t)et * a.ldy + en] = tt;
      if (a.stash) a.stash[(size_t)et * a.lds + en] = tt;
      if (a.out_planes) {
        const float gv = a.out_gain ? a.out_gain[en] * tt : tt;
        const uint32_t hi = f32_to_bf16(gv);
        a.out_planes[(size_t)et * a.out_ld + en] = (bf16_t)hi;
        a.out_planes[(size_t)(PR + et) * a.out_ld + en] = (bf16_t)f32_to_bf16(gv - bf16_to_f32(hi));
      }
      y2 = tt * tt;
    }
    if (a.out_ssq) {
      // the half tile's 8 features of row et: lanes et + 8 f of this wave
      y2 += __shfl_xor(y2, 8, SSD_WAVE);
      y2 += __shfl_xor(y2, 16, SSD_WAVE);
      y2 += __shfl_xor(y2, 32, SSD_WAVE);
      if (elive && lane < 8) a.out_ssq[(size_t)eh * PR + et] = y2;
    }
    return;
  }
  if (!ok) return;
  if (qkv) {
    if (ef < 4) {
      int m, c;
      qkv_tile(eh >> 1, m, c);
      qkv_store_pair(a, m, c + tile_row(eh & 1, ef), et, v0, sum_at(0, ef + 4));
    }
    return;
  }
  if (GATED) {
    const float act = apply_epi_act(a.epi, v0, sum_at(NB - 1, ef));
    if (a.y) a.y[(size_t)et * a.ldy + en] = act;
    if (a.out_planes) {
      const uint32_t hi = f32_to_bf16(act);
      a.out_planes[(size_t)et * a.out_ld + en] = (bf16_t)hi;
      a.out_planes[(size_t)(PR + et) * a.out_ld + en] = (bf16_t)f32_to_bf16(act - bf16_to_f32(hi));
    }
    return;
  }
  float* yp = a.y + (size_t)et * a.ldy + en;
  switch (a.epi) {
    case EPI_STORE: *yp = v0; break;
    case EPI_BIAS_GELU: *yp = gelu_tanh(v0 + a.bias[en]); break;
    case EPI_BIAS_RESID: *yp = (a.resid ? a.resid[(size_t)et * a.ldr + en] : 0.f) + (v0 + a.bias[en]); break;
    default: break;
  }
}

// Planes of gain * x and the row's sum of squares (ssq[m], one partial) for the first skinny
// launch of a pass — one block per row.
__global__ __launch_bounds__(256) void skinny_prep_kernel(const float* __restrict__ x, int ldx, int K,
                                                          const float* __restrict__ gain,
                                                          bf16_t* __restrict__ out, int ldo, int PR,
                                                          float* __restrict__ ssq) {
  __shared__ float red[4];
  const int m = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const float* xr = x + (size_t)m * ldx;
  float s2 = 0.f;
  for (int k = tid * 4; k < K; k += 1024) {
    const float4 v = *reinterpret_cast<const float4*>(xr + k);
    s2 += (v.x * v.x + v.y * v.y) + (v.z * v.z + v.w * v.w);
    const float4 g = gain ? *reinterpret_cast<const float4*>(gain + k) : make_float4(1.f, 1.f, 1.f, 1.f);
    const float f[4] = {v.x * g.x, v.y * g.y, v.z * g.z, v.w * g.w};
    uint32_t h[4], l[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      h[e] = f32_to_bf16(f[e]);
      l[e] = f32_to_bf16(f[e] - bf16_to_f32(h[e]));
    }
    *reinterpret_cast<uint2*>(out + (size_t)m * ldo + k) = make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16));
    *reinterpret_cast<uint2*>(out + (size_t)(PR + m) * ldo + k) = make_uint2(l[0] | (l[1] << 16), l[2] | (l[3] << 16));
  }
  s2 = wave_sum(s2);
  if (lane == 0) red[wave] = s2;
  __syncthreads();
  if (tid == 0) ssq[m] = (red[0] + red[1]) + (red[2] + red[3]);
}

// ---------------------------------------------------------------------------------------------
// MFMA tile path: 64x64 output tiles, K in steps of 64 staged through LDS.  The activations
// (normalised on the fly) are staged as bf16 hi / lo planes and each 16x16x32 step issues two
// MFMAs against the same weight fragment, so the products see near-fp32 inputs.
constexpr int TM = 64, TN = 64, TK = 64, TKP = TK + 8;

// Larger MFMA tiles for long row blocks (prefill): 128 rows x BN features per block, K in steps
// of 32, double-buffered in LDS.  The next step's inputs (RMS-normalised when RMS, then split into
// bf16 hi / lo planes) and weights are fetched into registers while the current step computes, so
// there is one barrier per step.  4 waves in a 2 x 2 grid, each 64 rows x BN/2 features of 16x16
// MFMA tiles.  Row statistics come from launch_row_stats.
constexpr int G2M = 128, G2K = 32, G2KP = G2K + 8;

template <bool GATED, int BN, bool RMS>
__global__ __launch_bounds__(256) void gemm2_kernel(const LinearArgs a) {
  constexpr int NB = GATED ? 2 : 1;
  constexpr int TJ = BN / 32;                // 16-wide feature tiles per wave
  constexpr int BTPR = 256 / BN;             // threads per weight row in staging
  constexpr int BKPT = G2K / BTPR;           // weight elements per thread and row
  constexpr int BQ = BKPT / 8;               // 16-byte pieces of them
  extern __shared__ __attribute__((aligned(16))) bf16_t g2s[];
  bf16_t* Ah = g2s;                                   // [2][G2M][G2KP]
  bf16_t* Al = Ah + 2 * G2M * G2KP;                   // [2][G2M][G2KP]
  bf16_t* Bs = Al + 2 * G2M * G2KP;                   // [2][NB][BN][G2KP]

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  // row tiles vary fastest: the blocks that share a weight tile run back to back and re-read it
  // from L2 / the Infinity Cache
  const int m0 = blockIdx.x * G2M, n0 = blockIdx.y * BN;
  const int K = a.K, M = a.M;
  const int n_out = GATED ? a.n_per : a.n_per * a.n_mats;
  const int mat = GATED ? 0 : n0 / a.n_per;  // tiles never straddle matrices (n_per % BN == 0)
  const int nbase = GATED ? n0 : n0 - mat * a.n_per;
  const bf16_t* w0 = reinterpret_cast<const bf16_t*>(GATED ? a.w[0] : (mat == 0 ? a.w[0] : (mat == 1 ? a.w[1] : a.w[2])));
  const bf16_t* w1 = reinterpret_cast<const bf16_t*>(a.w[1]);

  // staging roles: input row ar, 16 elements from ak; weight row br, BKPT elements from bk
  const int ar = tid >> 1, ak = (tid & 1) * 16;
  const int am = min(m0 + ar, M - 1);
  const bool arow = m0 + ar < M;
  const float rstd = RMS ? a.stats[am].y : 1.f;
  const int br = tid / BTPR, bk = (tid % BTPR) * BKPT;
  const int bn = min(nbase + br, a.n_per - 1);
  const float* xrow = a.x + (size_t)am * a.ldx + ak;
  const float* grow = a.gain + ak;
  const bf16_t* wrow0 = w0 + (size_t)bn * K + bk;
  const bf16_t* wrow1 = w1 + (size_t)bn * K + bk;

  f32x4_t acc[NB][4][TJ];
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < TJ; ++j) acc[b][i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const int nk = K / G2K;
  const int kk = (lane >> 4) * 8;
  // kt = -1 only stages step 0
  for (int kt = -1; kt < nk; ++kt) {
    const bool next = kt + 1 < nk;
    // the next step's operands (the last step re-reads its own: unconditional loads keep them in
    // registers)
    float4 xa[4], ga[4];
    uint4 wa[BQ], wg[BQ];
    {
      const int k0 = min(kt + 1, nk - 1) * G2K;
#pragma unroll
      for (int q = 0; q < 4; ++q) xa[q] = reinterpret_cast<const float4*>(xrow + k0)[q];
#pragma unroll
      for (int q = 0; q < BQ; ++q) wa[q] = reinterpret_cast<const uint4*>(wrow0 + k0)[q];
#pragma unroll
      for (int q = 0; q < BQ; ++q) wg[q] = GATED ? reinterpret_cast<const uint4*>(wrow1 + k0)[q] : wa[q];
#pragma unroll
      for (int q = 0; q < 4; ++q) ga[q] = RMS ? reinterpret_cast<const float4*>(grow + k0)[q] : xa[q];
    }
    if (kt >= 0) {
      const int buf = kt & 1;
      bf16x8_t fh[4], fl[4], fb[NB][TJ];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const size_t r = ((size_t)buf * G2M + wm * 64 + 16 * i + (lane & 15)) * G2KP + kk;
        fh[i] = *reinterpret_cast<const bf16x8_t*>(Ah + r);
        fl[i] = *reinterpret_cast<const bf16x8_t*>(Al + r);
      }
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int j = 0; j < TJ; ++j)
          fb[b][j] = *reinterpret_cast<const bf16x8_t*>(
              Bs + (((size_t)buf * NB + b) * BN + wn * (BN / 2) + 16 * j + (lane & 15)) * G2KP + kk);
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < TJ; ++j) {
            acc[b][i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fh[i], fb[b][j], acc[b][i][j], 0, 0, 0);
            acc[b][i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fl[i], fb[b][j], acc[b][i][j], 0, 0, 0);
          }
    }
    if (next) {
      const int buf = (kt + 1) & 1;
      float f[16];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float4 v = xa[q];
        if (RMS) {
          v.x *= rstd * ga[q].x; v.y *= rstd * ga[q].y; v.z *= rstd * ga[q].z; v.w *= rstd * ga[q].w;
        }
        f[4 * q] = arow ? v.x : 0.f;
        f[4 * q + 1] = arow ? v.y : 0.f;
        f[4 * q + 2] = arow ? v.z : 0.f;
        f[4 * q + 3] = arow ? v.w : 0.f;
      }
      uint4 h0, l0, h1, l1;
      split_bf16x8(f, h0, l0);
      split_bf16x8(f + 8, h1, l1);
      uint4* ah = reinterpret_cast<uint4*>(Ah + ((size_t)buf * G2M + ar) * G2KP + ak);
      uint4* al = reinterpret_cast<uint4*>(Al + ((size_t)buf * G2M + ar) * G2KP + ak);
      ah[0] = h0;
      ah[1] = h1;
      al[0] = l0;
      al[1] = l1;
      uint4* bp = reinterpret_cast<uint4*>(Bs + (((size_t)buf * NB) * BN + br) * G2KP + bk);
#pragma unroll
      for (int q = 0; q < BQ; ++q) bp[q] = wa[q];
      if (GATED) {
        uint4* bq = reinterpret_cast<uint4*>(Bs + (((size_t)buf * NB + 1) * BN + br) * G2KP + bk);
#pragma unroll
        for (int q = 0; q < BQ; ++q) bq[q] = wg[q];
      }
    }
    __syncthreads();
  }

  // epilogue: lane holds D[4 * (lane / 16) + e][lane % 16] of each 16x16 tile
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < TJ; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int m = m0 + wm * 64 + 16 * i + 4 * (lane >> 4) + e;
        const int n = n0 + wn * (BN / 2) + 16 * j + (lane & 15);
        if (m >= M || n >= n_out) continue;
        const float v = acc[0][i][j][e];
        float* yp = a.y + (size_t)m * a.ldy + n;
        if (GATED) {
          *yp = apply_epi_act(a.epi, v, acc[NB - 1][i][j][e]);
          continue;
        }
        switch (a.epi) {
          case EPI_STORE: *yp = v; break;
          case EPI_RESID: {
            const float t = *yp + v;
            *yp = t;
            if (a.stash) a.stash[(size_t)m * a.lds + n] = t;
            break;
          }
          case EPI_BIAS_GELU: *yp = gelu_tanh(v + a.bias[n]); break;
          case EPI_BIAS_RESID: *yp = (a.resid ? a.resid[(size_t)m * a.ldr + n] : 0.f) + (v + a.bias[n]); break;
          default: break;
        }
      }
}

// Prefill GEMM on bf16 operand planes: the input rows arrive as hi / lo planes of g * x written
// once by plane_prep_kernel (which also leaves 1/rms of each row in stats[m].y), so a K step
// stages bf16 only and nothing is re-normalised per column tile.  A block owns TMR rows x BN
// features (x2 matrices when gated) on a 2 x 2 grid of waves; K advances in steps of 32 through
// double-buffered LDS (one barrier a step), and each thread keeps the global loads of the next D
// steps in flight in a rotating set of registers, so a step's memory round trip overlaps D steps
// of MFMA work instead of one.  RMSNorm scales the outputs by 1/rms.
constexpr int G3K = 32, G3KP = G3K + 8, G3D = 4;  // G3D: the slot code below assumes 4

template <bool GATED, int TMR, int BN, bool RMS>
__global__ __launch_bounds__(256, 2) void gemm3_kernel(const LinearArgs a) {
  constexpr int NB = GATED ? 2 : 1;
  constexpr int IF = TMR / 32;        // 16-row fragments per wave (the wave covers TMR / 2 rows)
  constexpr int TJ = BN / 32;         // 16-feature fragments per wave (BN / 2 features)
  constexpr int AQ = TMR / 64;        // 16-byte pieces of each plane a thread stages per step
  constexpr int BQ = BN / 64;         // 16-byte pieces of each weight matrix a thread stages
  constexpr int ATPR = 256 / TMR;     // threads per input row in staging
  constexpr int BTPR = 256 / BN;      // threads per weight row in staging
  extern __shared__ __attribute__((aligned(16))) bf16_t g3s[];
  bf16_t* Ah = g3s;                          // [2][TMR][G3KP]
  bf16_t* Al = Ah + 2 * TMR * G3KP;          // [2][TMR][G3KP]
  bf16_t* Bs = Al + 2 * TMR * G3KP;          // [2][NB][BN][G3KP]

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  // Tile of this block.  Workgroups are dealt to the 8 XCDs round-robin by linear id, and each
  // XCD has its own L2, so the linear id is mapped to a contiguous range of tiles per XCD
  // (row tiles fastest, then K ranges, then weight tiles): the blocks that share a weight tile,
  // or a range of the input planes, run on one XCD and read it through one L2.
  int rt, zs, ct;
  {
    const int nx = gridDim.x, nz = gridDim.z, T = nx * gridDim.y * nz;
    const int id = blockIdx.x + nx * (blockIdx.y + gridDim.y * blockIdx.z);
    const int xcd = id & 7, slot = id >> 3;
    const int t = xcd * (T >> 3) + min(xcd, T & 7) + slot;
    rt = t % nx;
    const int rest = t / nx;
    zs = rest % nz;
    ct = rest / nz;
  }
  const int m0 = rt * TMR, n0 = ct * BN;
  const int K = a.K, M = a.M;
  // K range of this block: all of K, or range zs of a.ksplit (whole steps each)
  int nk = K / G3K, kb = 0;
  if (!GATED && a.ksplit > 1) {
    const int per = (nk + a.ksplit - 1) / a.ksplit;
    kb = zs * per * G3K;
    nk = min(per, nk - zs * per);
  }
  const int n_out = GATED ? a.n_per : a.n_per * a.n_mats;
  const int mat = GATED ? 0 : n0 / a.n_per;  // tiles never straddle matrices (n_per % BN == 0)
  const int nbase = GATED ? n0 : n0 - mat * a.n_per;
  const bf16_t* w0 = reinterpret_cast<const bf16_t*>(GATED ? a.w[0] : (mat == 0 ? a.w[0] : (mat == 1 ? a.w[1] : a.w[2])));
  const bf16_t* w1 = reinterpret_cast<const bf16_t*>(a.w[1]);

  // staging roles: input row ar (clamped: rows past M are computed and never stored), AQ * 8
  // elements from ak; weight row br, BQ * 8 elements from bk
  const int ar = tid / ATPR, ak = (tid % ATPR) * (AQ * 8);
  const int br = tid / BTPR, bk = (tid % BTPR) * (BQ * 8);
  const bf16_t* hrow = a.in_planes + (size_t)min(m0 + ar, M - 1) * a.in_ld + kb + ak;
  const bf16_t* lrow = hrow + (size_t)a.plane_rows * a.in_ld;
  const int bn = min(nbase + br, a.n_per - 1);
  const bf16_t* wrow0 = w0 + (size_t)bn * K + kb + bk;
  const bf16_t* wrow1 = w1 + (size_t)bn * K + kb + bk;

  f32x4_t acc[NB][IF][TJ];
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int i = 0; i < IF; ++i)
#pragma unroll
      for (int j = 0; j < TJ; ++j) acc[b][i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
  u32x4_t rh[G3D][AQ], rl[G3D][AQ], rw[G3D][NB][BQ];
  // (macros, so that every slot index is a constant and the ring stays in registers)
#define G3_FETCH(SLOT, STEP)                                                               \
  do {                                                                                     \
    const int k0_ = min((STEP), nk - 1) * G3K;                                             \
    _Pragma("unroll") for (int q = 0; q < AQ; ++q) {                                       \
      rh[SLOT][q] = reinterpret_cast<const u32x4_t*>(hrow + k0_)[q];                         \
      rl[SLOT][q] = reinterpret_cast<const u32x4_t*>(lrow + k0_)[q];                         \
    }                                                                                      \
    _Pragma("unroll") for (int q = 0; q < BQ; ++q) {                                       \
      rw[SLOT][0][q] = reinterpret_cast<const u32x4_t*>(wrow0 + k0_)[q];                     \
      if (GATED) rw[SLOT][NB - 1][q] = reinterpret_cast<const u32x4_t*>(wrow1 + k0_)[q];     \
    }                                                                                      \
  } while (0)
#define G3_STAGE(SLOT, BUF)                                                                \
  do {                                                                                     \
    u32x4_t* ah_ = reinterpret_cast<u32x4_t*>(Ah + ((size_t)(BUF) * TMR + ar) * G3KP + ak);    \
    u32x4_t* al_ = reinterpret_cast<u32x4_t*>(Al + ((size_t)(BUF) * TMR + ar) * G3KP + ak);    \
    _Pragma("unroll") for (int q = 0; q < AQ; ++q) {                                       \
      ah_[q] = rh[SLOT][q];                                                                \
      al_[q] = rl[SLOT][q];                                                                \
    }                                                                                      \
    _Pragma("unroll") for (int b = 0; b < NB; ++b) {                                       \
      u32x4_t* bp_ = reinterpret_cast<u32x4_t*>(Bs + (((size_t)(BUF) * NB + b) * BN + br) * G3KP + bk); \
      _Pragma("unroll") for (int q = 0; q < BQ; ++q) bp_[q] = rw[SLOT][b][q];              \
    }                                                                                      \
  } while (0)

  // prologue: steps 0..D-1 in flight, step 0 staged
  G3_FETCH(0, 0);
  G3_FETCH(1, 1);
  G3_FETCH(2, 2);
  G3_FETCH(3, 3);
  G3_STAGE(0, 0);
  G3_FETCH(0, G3D);
  __syncthreads();

  const int kk = (lane >> 4) * 8;
  // one K step: MFMAs on LDS buffer step & 1, then slot NEXT (holding step + 1) staged into the
  // other buffer and refilled with step + 1 + D; unrolled by hand over the four slots (a loop
  // with a barrier in its body is not unrolled, and a variable slot would put the ring in memory)
#define G3_BODY(NEXT)                                                                      \
  if (step < nk) {                                                                         \
    const int buf = step & 1;                                                              \
    bf16x8_t fh[IF], fl[IF], fb[NB][TJ];                                                   \
    _Pragma("unroll") for (int i = 0; i < IF; ++i) {                                       \
      const size_t r = ((size_t)buf * TMR + wm * (TMR / 2) + 16 * i + (lane & 15)) * G3KP + kk; \
      fh[i] = *reinterpret_cast<const bf16x8_t*>(Ah + r);                                  \
      fl[i] = *reinterpret_cast<const bf16x8_t*>(Al + r);                                  \
    }                                                                                      \
    _Pragma("unroll") for (int b = 0; b < NB; ++b)                                         \
    _Pragma("unroll") for (int j = 0; j < TJ; ++j)                                         \
      fb[b][j] = *reinterpret_cast<const bf16x8_t*>(                                       \
          Bs + (((size_t)buf * NB + b) * BN + wn * (BN / 2) + 16 * j + (lane & 15)) * G3KP + kk); \
    _Pragma("unroll") for (int b = 0; b < NB; ++b)                                         \
    _Pragma("unroll") for (int i = 0; i < IF; ++i)                                         \
    _Pragma("unroll") for (int j = 0; j < TJ; ++j) {                                       \
      acc[b][i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fh[i], fb[b][j], acc[b][i][j], 0, 0, 0); \
      acc[b][i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fl[i], fb[b][j], acc[b][i][j], 0, 0, 0); \
    }                                                                                      \
    if (step + 1 < nk) {                                                                   \
      G3_STAGE(NEXT, buf ^ 1);                                                             \
      G3_FETCH(NEXT, step + 1 + G3D);                                                      \
    }                                                                                      \
    __syncthreads();                                                                       \
  }
  // Full groups of four steps whose next step exists run as straight-line code: with no branch
  // between them the compiler can wait for just the slot it stages (a branch would make it wait
  // for every load in flight, the whole ring).  The last group takes the guarded bodies.
#define G3_BODY_U(NEXT)                                                                    \
  {                                                                                        \
    const int buf = step & 1;                                                              \
    bf16x8_t fh[IF], fl[IF], fb[NB][TJ];                                                   \
    _Pragma("unroll") for (int i = 0; i < IF; ++i) {                                       \
      const size_t r = ((size_t)buf * TMR + wm * (TMR / 2) + 16 * i + (lane & 15)) * G3KP + kk; \
      fh[i] = *reinterpret_cast<const bf16x8_t*>(Ah + r);                                  \
      fl[i] = *reinterpret_cast<const bf16x8_t*>(Al + r);                                  \
    }                                                                                      \
    _Pragma("unroll") for (int b = 0; b < NB; ++b)                                         \
    _Pragma("unroll") for (int j = 0; j < TJ; ++j)                                         \
      fb[b][j] = *reinterpret_cast<const bf16x8_t*>(                                       \
          Bs + (((size_t)buf * NB + b) * BN + wn * (BN / 2) + 16 * j + (lane & 15)) * G3KP + kk); \
    _Pragma("unroll") for (int b = 0; b < NB; ++b)                                         \
    _Pragma("unroll") for (int i = 0; i < IF; ++i)                                         \
    _Pragma("unroll") for (int j = 0; j < TJ; ++j) {                                       \
      acc[b][i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fh[i], fb[b][j], acc[b][i][j], 0, 0, 0); \
      acc[b][i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fl[i], fb[b][j], acc[b][i][j], 0, 0, 0); \
    }                                                                                      \
    G3_STAGE(NEXT, buf ^ 1);                                                               \
    G3_FETCH(NEXT, step + 1 + G3D);                                                        \
    __syncthreads();                                                                       \
  }
  int kt = 0;
  for (; kt + G3D < nk; kt += G3D) {
    int step = kt;
    G3_BODY_U(1)
    step = kt + 1;
    G3_BODY_U(2)
    step = kt + 2;
    G3_BODY_U(3)
    step = kt + 3;
    G3_BODY_U(0)
  }
  {
    int step = kt;
    G3_BODY(1)
    step = kt + 1;
    G3_BODY(2)
    step = kt + 2;
    G3_BODY(3)
    step = kt + 3;
    G3_BODY(0)
  }
#undef G3_BODY_U
#undef G3_BODY

  // epilogue: lane holds D[4 * (lane / 16) + e][lane % 16] of each 16x16 tile
#pragma unroll
  for (int i = 0; i < IF; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int m = m0 + wm * (TMR / 2) + 16 * i + 4 * (lane >> 4) + e;
      if (m >= M) continue;
      const float rsc = RMS ? a.stats[m].y : 1.f;
#pragma unroll
      for (int j = 0; j < TJ; ++j) {
        const int n = n0 + wn * (BN / 2) + 16 * j + (lane & 15);
        if (n >= n_out) continue;
        const float v = acc[0][i][j][e] * rsc;
        if (!GATED && a.ksplit > 1) {
          a.kpart[((size_t)zs * a.gemm_plane_rows + m) * a.kpart_ld + n] = v;
          continue;
        }
        float* yp = a.y + (size_t)m * a.ldy + n;
        if (GATED) {
          *yp = apply_epi_act(a.epi, v, acc[NB - 1][i][j][e] * rsc);
          continue;
        }
        switch (a.epi) {
          case EPI_STORE: *yp = v; break;
          case EPI_RESID: {
            const float t = *yp + v;
            *yp = t;
            if (a.stash) a.stash[(size_t)m * a.lds + n] = t;
            break;
          }
          case EPI_BIAS_GELU: *yp = gelu_tanh(v + a.bias[n]); break;
          case EPI_BIAS_RESID: *yp = (a.resid ? a.resid[(size_t)m * a.ldr + n] : 0.f) + (v + a.bias[n]); break;
          default: break;
        }
      }
    }
}

#undef G3_FETCH
#undef G3_STAGE

// Planes of g * x (g = gain, or 1) for rows 0..M-1 and, with a gain (RMSNorm), 1/rms of each row
// in stats[m].y; one block per row.  hi of row m at out + m * ldo, lo plane_rows rows later.
__global__ __launch_bounds__(256) void plane_prep_kernel(const float* __restrict__ x, int ldx, int K,
                                                         const float* __restrict__ gain, float eps,
                                                         bf16_t* __restrict__ out, int ldo,
                                                         int plane_rows, float2* __restrict__ stats) {
  __shared__ float red[4];
  const int m = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const float* xr = x + (size_t)m * ldx;
  float s2 = 0.f;
  for (int k = tid * 8; k < K; k += 2048) {
    float f[8];
    const float4 v0 = *reinterpret_cast<const float4*>(xr + k);
    const float4 v1 = *reinterpret_cast<const float4*>(xr + k + 4);
    f[0] = v0.x; f[1] = v0.y; f[2] = v0.z; f[3] = v0.w; f[4] = v1.x; f[5] = v1.y; f[6] = v1.z; f[7] = v1.w;
#pragma unroll
    for (int e = 0; e < 8; ++e) s2 = fmaf(f[e], f[e], s2);
    if (gain) {
      const float4 g0 = *reinterpret_cast<const float4*>(gain + k);
      const float4 g1 = *reinterpret_cast<const float4*>(gain + k + 4);
      f[0] *= g0.x; f[1] *= g0.y; f[2] *= g0.z; f[3] *= g0.w;
      f[4] *= g1.x; f[5] *= g1.y; f[6] *= g1.z; f[7] *= g1.w;
    }
    uint4 h, l;
    split_bf16x8(f, h, l);
    *reinterpret_cast<uint4*>(out + (size_t)m * ldo + k) = h;
    *reinterpret_cast<uint4*>(out + (size_t)(plane_rows + m) * ldo + k) = l;
  }
  if (!gain) return;
  s2 = wave_sum(s2);
  if (lane == 0) red[wave] = s2;
  __syncthreads();
  if (tid == 0) stats[m] = make_float2(0.f, 1.0f / sqrtf(((red[0] + red[1]) + (red[2] + red[3])) / (float)K + eps));
}

// y[m][n] += (p_0 + p_1 + ... + p_{S-1})[m][n] over the K-range partials of the tile path, added
// in range order (the stash, when set, receives the new y too); four outputs per thread.
__global__ __launch_bounds__(256) void ksum_kernel(const LinearArgs a, int n_out) {
  const int q = blockIdx.x * 256 + threadIdx.x;  // float4 index over M x n_out
  const int per_row = n_out >> 2;
  if (q >= a.M * per_row) return;
  const int m = q / per_row, n = (q - m * per_row) * 4;
  float4 p[4];
#pragma unroll
  for (int s = 0; s < 4; ++s)
    if (s < a.ksplit)
      p[s] = *reinterpret_cast<const float4*>(a.kpart + ((size_t)s * a.gemm_plane_rows + m) * a.kpart_ld + n);
  float4 t = p[0];
#pragma unroll
  for (int s = 1; s < 4; ++s)
    if (s < a.ksplit) { t.x += p[s].x; t.y += p[s].y; t.z += p[s].z; t.w += p[s].w; }
  float4* yp = reinterpret_cast<float4*>(a.y + (size_t)m * a.ldy + n);
  float4 y = *yp;
  y.x += t.x; y.y += t.y; y.z += t.z; y.w += t.w;
  *yp = y;
  if (a.stash) *reinterpret_cast<float4*>(a.stash + (size_t)m * a.lds + n) = y;
}

template <bool GATED>
__global__ __launch_bounds__(256) void gemm_kernel(const LinearArgs a) {
  constexpr int NB = GATED ? 2 : 1;
  __shared__ __attribute__((aligned(16))) bf16_t As[2][TM][TKP];  // hi, lo planes
  __shared__ __attribute__((aligned(16))) bf16_t Bs[NB][TN][TKP];
  __shared__ float am_v[TM][TN / 16];
  __shared__ int am_i[TM][TN / 16];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int m0 = blockIdx.y * TM, n0 = blockIdx.x * TN;
  const int wm = (wave >> 1) * 32, wn = (wave & 1) * 32;
  const int K = a.K;
  const int n_out = GATED ? a.n_per : a.n_per * a.n_mats;
  const int mat = GATED ? 0 : n0 / a.n_per;  // tiles never straddle matrices (n_per % 64 == 0)
  const int nbase = GATED ? n0 : n0 - mat * a.n_per;
  const bf16_t* W0 = reinterpret_cast<const bf16_t*>(GATED ? a.w[0] : (mat == 0 ? a.w[0] : (mat == 1 ? a.w[1] : a.w[2])));
  const bf16_t* W1 = reinterpret_cast<const bf16_t*>(a.w[1]);

  f32x4_t acc[NB][2][2];
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[b][i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const int lr = tid >> 2, lk = (tid & 3) * 16;  // staging: row, 16-element column group
  const int am = m0 + lr;
  const bool arow = am < a.M;
  float2 stat = make_float2(0.f, 1.f);
  if (arow && a.norm != NORM_NONE) stat = a.stats[am];
  const int wrow = nbase + lr;
  const bool brow = (n0 + lr) < n_out;

  for (int k0 = 0; k0 < K; k0 += TK) {
    float f[16];
    if (arow) {
      const float* xp = a.x + (size_t)am * a.ldx + k0 + lk;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float4 v = reinterpret_cast<const float4*>(xp)[q];
        f[4 * q] = v.x; f[4 * q + 1] = v.y; f[4 * q + 2] = v.z; f[4 * q + 3] = v.w;
      }
      if (a.norm != NORM_NONE) {
#pragma unroll
        for (int q = 0; q < 16; ++q) {
          f[q] = (f[q] - stat.x) * stat.y * a.gain[k0 + lk + q];
          if (a.norm == NORM_LN) f[q] += a.shift[k0 + lk + q];
        }
      }
    } else {
#pragma unroll
      for (int q = 0; q < 16; ++q) f[q] = 0.f;
    }
    uint4 pa0, pa1, pl0, pl1;
    split_bf16x8(f, pa0, pl0);
    split_bf16x8(f + 8, pa1, pl1);
    uint4 pb[NB][2];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      if (brow) {
        const bf16_t* wp = (b == 0 ? W0 : W1) + (size_t)wrow * K + k0 + lk;
        pb[b][0] = reinterpret_cast<const uint4*>(wp)[0];
        pb[b][1] = reinterpret_cast<const uint4*>(wp)[1];
      } else {
        pb[b][0] = pb[b][1] = make_uint4(0, 0, 0, 0);
      }
    }
    __syncthreads();
    *reinterpret_cast<uint4*>(&As[0][lr][lk]) = pa0;
    *reinterpret_cast<uint4*>(&As[0][lr][lk + 8]) = pa1;
    *reinterpret_cast<uint4*>(&As[1][lr][lk]) = pl0;
    *reinterpret_cast<uint4*>(&As[1][lr][lk + 8]) = pl1;
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      *reinterpret_cast<uint4*>(&Bs[b][lr][lk]) = pb[b][0];
      *reinterpret_cast<uint4*>(&Bs[b][lr][lk + 8]) = pb[b][1];
    }
    __syncthreads();
#pragma unroll
    for (int ks = 0; ks < TK; ks += 32) {
      const int kk = ks + (lane >> 4) * 8;
      bf16x8_t af[2][2], bfr[NB][2];
#pragma unroll
      for (int pl = 0; pl < 2; ++pl)
#pragma unroll
        for (int i = 0; i < 2; ++i)
          af[pl][i] = *reinterpret_cast<const bf16x8_t*>(&As[pl][wm + 16 * i + (lane & 15)][kk]);
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          bfr[b][j] = *reinterpret_cast<const bf16x8_t*>(&Bs[b][wn + 16 * j + (lane & 15)][kk]);
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j) {
            acc[b][i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[0][i], bfr[b][j], acc[b][i][j], 0, 0, 0);
            acc[b][i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[1][i], bfr[b][j], acc[b][i][j], 0, 0, 0);
          }
    }
  }

  if (!GATED && a.epi == EPI_ARGMAX) {
    // per row of the tile: best over this thread's columns, then over the 64 columns
    float bv[2][4];
    int bi[2][4];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        bv[i][e] = -INFINITY;
        bi[i][e] = INT_MAX;
        const int m = m0 + wm + 16 * i + 4 * (lane >> 4) + e;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int n = n0 + wn + 16 * j + (lane & 15);
          if (n < n_out && m < a.M) {
            argmax_merge(bv[i][e], bi[i][e], acc[0][i][j][e], n);
            if (a.logits) a.logits[(size_t)m * a.ldl + n] = acc[0][i][j][e];
          }
        }
      }
    // reduce across the 16 lanes that share rows (lane & 15 varies)
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
#pragma unroll
        for (int o = 8; o > 0; o >>= 1) {
          const float v2 = __shfl_xor(bv[i][e], o, SSD_WAVE);
          const int i2 = __shfl_xor(bi[i][e], o, SSD_WAVE);
          argmax_merge(bv[i][e], bi[i][e], v2, i2);
        }
        if ((lane & 15) == 0) {
          const int ml = wm + 16 * i + 4 * (lane >> 4) + e;
          am_v[ml][wn / 16] = bv[i][e];
          am_i[ml][wn / 16] = bi[i][e];
          am_v[ml][wn / 16 + 1] = -INFINITY;
          am_i[ml][wn / 16 + 1] = INT_MAX;
        }
      }
    __syncthreads();
    if (tid < TM && m0 + tid < a.M) {
      float v = -INFINITY;
      int i = INT_MAX;
      for (int c = 0; c < TN / 16; ++c) argmax_merge(v, i, am_v[tid][c], am_i[tid][c]);
      a.part_val[(size_t)(m0 + tid) * a.n_parts + blockIdx.x] = v;
      a.part_idx[(size_t)(m0 + tid) * a.n_parts + blockIdx.x] = i;
    }
    return;
  }

#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int m = m0 + wm + 16 * i + 4 * (lane >> 4) + e;
        const int n = n0 + wn + 16 * j + (lane & 15);
        if (m >= a.M || n >= n_out) continue;
        float* yp = a.y + (size_t)m * a.ldy + n;
        const float v = acc[0][i][j][e];
        if (GATED) {
          *yp = apply_epi_act(a.epi, v, acc[NB - 1][i][j][e]);
          continue;
        }
        switch (a.epi) {
          case EPI_STORE: *yp = v; break;
          case EPI_RESID: {
            const float t = *yp + v;
            *yp = t;
            if (a.stash) a.stash[(size_t)m * a.lds + n] = t;
            break;
          }
          case EPI_BIAS_GELU: *yp = gelu_tanh(v + a.bias[n]); break;
          case EPI_BIAS_RESID:
            *yp = (a.resid ? a.resid[(size_t)m * a.ldr + n] : 0.f) + (v + a.bias[n]);
            break;
          default: break;
        }
      }
}

__global__ void row_stats_kernel(const float* x, int ldx, int M, int K, int norm, float eps,
                                 float2* stats) {
  const int m = blockIdx.x;
  if (m >= M) return;
  const int lane = threadIdx.x;  // one wave
  const float* xr = x + (size_t)m * ldx;
  float mean = 0.f;
  if (norm == NORM_LN) {
    float s1 = 0.f;
    for (int k = lane; k < K; k += 64) s1 += xr[k];
    mean = wave_sum(s1) / (float)K;
  }
  float s2 = 0.f;
  for (int k = lane; k < K; k += 64) {
    const float t = xr[k] - mean;
    s2 += t * t;
  }
  s2 = wave_sum(s2);
  if (lane == 0) stats[m] = make_float2(mean, 1.0f / sqrtf(s2 / (float)K + eps));
}

int device_cus() {
  static int cus = 0;
  if (!cus) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus <= 0)
      cus = 256;
  }
  return cus;
}

// Vector-path launch shape: MB input rows per block (grid.y = row blocks), blocks over row groups.
struct GvPlan {
  int mb, blocks;
};

GvPlan gv_plan(const LinearArgs& a) {
  GvPlan p;
  const int kpad = (a.K + 7) & ~7;
  int mb = a.M < 1 ? 1 : (a.M > 8 ? 8 : a.M);
  while (mb > 1 && mb * kpad > GV_LDS_FLOATS) --mb;
  p.mb = mb;
  const bool gated = (a.epi == EPI_GATED_GELU || a.epi == EPI_GATED_SILU);
  const int n_total = gated ? a.n_per : a.n_per * a.n_mats;
  const int n_pairs = gated ? a.n_per : (n_total + 1) / 2;
  const int groups = (n_pairs + GV_WAVES - 1) / GV_WAVES;
  p.blocks = groups;
  return p;
}

template <typename WT, int KP, int NORM>
void launch_gemv1(const LinearArgs& a, dim3 grid, hipStream_t s, LaunchTiming* t) {
  if (t) {
    hipExtLaunchKernelGGL((gemv1_kernel<WT, KP, NORM>), grid, dim3(256), 0u, s, t->start, t->stop,
                          0u, a);
    t->timed = true;
  } else {
    hipLaunchKernelGGL((gemv1_kernel<WT, KP, NORM>), grid, dim3(256), 0, s, a);
  }
}

template <int KP, int NORM, typename WT = bf16_t>
void launch_gemv1k(const LinearArgs& a, dim3 grid, hipStream_t s, LaunchTiming* t) {
  if (t) {
    hipExtLaunchKernelGGL((gemv1k_kernel<WT, KP, NORM>), grid, dim3(256), 0u, s, t->start,
                          t->stop, 0u, a);
    t->timed = true;
  } else {
    hipLaunchKernelGGL((gemv1k_kernel<WT, KP, NORM>), grid, dim3(256), 0, s, a);
  }
}

// One bf16 row with 2048 <= K <= 6144 and no LayerNorm, or up to 12288 without a norm (the
// LLaMA-7B down projection, K = 11008): the K-split kernel (same grid as gemv1).  float32
// weights at K = 2048 too (the folded cross-attention scores of a FlanT5-xl-sized layer).
bool use_gemv1k(const LinearArgs& a) {
  if (a.M != 1 || a.K < 2048 || a.K % 8) return false;
  if (a.wdtype != 1) return a.K == 2048 && (a.norm == NORM_RMS || a.norm == NORM_NONE);
  if (a.norm == NORM_RMS) return a.K <= 3 * 2048;
  return a.norm == NORM_NONE && a.K <= 6 * 2048;
}

hipError_t launch_gemv1k_any(const LinearArgs& a, hipStream_t s, LaunchTiming* t) {
  const dim3 grid(gv_plan(a).blocks);
  const bool timed = t && a.K == t->K && a.norm == t->norm && a.wdtype == t->wdtype && t->start &&
                     t->stop;
  LaunchTiming* tt = timed ? t : nullptr;
  const int kp = (a.K + 2047) / 2048;
  const bool rms = a.norm == NORM_RMS;
  if (a.wdtype != 1) {
    rms ? launch_gemv1k<1, NORM_RMS, float>(a, grid, s, tt)
        : launch_gemv1k<1, NORM_NONE, float>(a, grid, s, tt);
  } else if (kp == 1) rms ? launch_gemv1k<1, NORM_RMS>(a, grid, s, tt) : launch_gemv1k<1, NORM_NONE>(a, grid, s, tt);
  else if (kp == 2) rms ? launch_gemv1k<2, NORM_RMS>(a, grid, s, tt) : launch_gemv1k<2, NORM_NONE>(a, grid, s, tt);
  else if (kp == 3) rms ? launch_gemv1k<3, NORM_RMS>(a, grid, s, tt) : launch_gemv1k<3, NORM_NONE>(a, grid, s, tt);
  else if (kp == 4) launch_gemv1k<4, NORM_NONE>(a, grid, s, tt);
  else if (kp == 5) launch_gemv1k<5, NORM_NONE>(a, grid, s, tt);
  else launch_gemv1k<6, NORM_NONE>(a, grid, s, tt);
  return hipGetLastError();
}

template <typename WT, int MB, int KP>
hipError_t launch_gemv_kp(const LinearArgs& a, const GvPlan& p, hipStream_t s, LaunchTiming* t) {
  static bool attr = false;
  if (!attr) {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&gemv_kernel<WT, MB, KP>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, GV_LDS_FLOATS * 4);
    attr = true;
  }
  dim3 grid(p.blocks, (a.M + MB - 1) / MB);
  if (MB == 1 && a.M == 1 && (a.norm == NORM_LN ? a.K <= 2048 : a.K <= 512 * KP)) {
    // one row that fits a batch: the register path
    const bool timed = t && a.K == t->K && a.norm == t->norm &&
                       (int)(sizeof(WT) == 2) == t->wdtype && t->start && t->stop;
    if (a.norm == NORM_RMS) launch_gemv1<WT, KP, NORM_RMS>(a, grid, s, timed ? t : nullptr);
    else if (a.norm == NORM_LN) launch_gemv1<WT, 4, NORM_LN>(a, grid, s, timed ? t : nullptr);
    else if (a.norm == NORM_SOFTMAX) launch_gemv1<WT, KP, NORM_SOFTMAX>(a, grid, s, nullptr);
    else launch_gemv1<WT, KP, NORM_NONE>(a, grid, s, timed ? t : nullptr);
    return hipGetLastError();
  }
  if (a.norm == NORM_SOFTMAX) return hipErrorInvalidValue;
  const size_t shm = (size_t)MB * ((a.K + 7) & ~7) * sizeof(float);
  hipLaunchKernelGGL((gemv_kernel<WT, MB, KP>), grid, dim3(256), shm, s, a);
  return hipGetLastError();
}

}  // namespace

// whole rows up to 12 pieces of 512 elements (6144) in one batch (2 or 4 pieces for short rows),
// else batches of 8
int gemv_pieces(int K) {
  const int pieces = (K + 511) / 512;
  if (pieces <= 2) return 2;
  if (pieces <= 4) return 4;
  if (pieces <= 8 || pieces > 12) return 8;
  return 12;
}

namespace {

template <typename WT, int MB>
hipError_t launch_gemv_mb(const LinearArgs& a, const GvPlan& p, hipStream_t s, LaunchTiming* t) {
  switch (gemv_pieces(a.K)) {
    case 2: return launch_gemv_kp<WT, MB, 2>(a, p, s, t);
    case 4: return launch_gemv_kp<WT, MB, 4>(a, p, s, t);
    case 12: return launch_gemv_kp<WT, MB, 12>(a, p, s, t);
    default: return launch_gemv_kp<WT, MB, 8>(a, p, s, t);
  }
}

template <typename WT>
hipError_t launch_gemv_t(const LinearArgs& a, hipStream_t s, LaunchTiming* t) {
  const GvPlan p = gv_plan(a);
  switch (p.mb) {
    case 1: return launch_gemv_mb<WT, 1>(a, p, s, t);
    case 2: return launch_gemv_mb<WT, 2>(a, p, s, t);
    case 3: return launch_gemv_mb<WT, 3>(a, p, s, t);
    case 4: return launch_gemv_mb<WT, 4>(a, p, s, t);
    case 5: return launch_gemv_mb<WT, 5>(a, p, s, t);
    case 6: return launch_gemv_mb<WT, 6>(a, p, s, t);
    case 7: return launch_gemv_mb<WT, 7>(a, p, s, t);
    default: return launch_gemv_mb<WT, 8>(a, p, s, t);
  }
}

bool want_mfma(const LinearArgs& a) {
  if (a.wdtype != 1) return false;
  if (a.K % TK) return false;
  if (a.n_mats > 1 && a.n_per % TN) return false;  // tiles must not straddle matrices
  if (a.use_mfma >= 0) return a.use_mfma == 1;
  return a.M > 8;
}

}  // namespace

bool linear_pair_ok(const LinearArgs& a, const LinearArgs& b) {
  auto plain = [](const LinearArgs& x) {
    return x.M == 1 && x.norm == NORM_NONE && x.K >= 8 && x.K % 8 == 0 &&
           (x.epi == EPI_STORE || x.epi == EPI_RESID || x.epi == EPI_BIAS_RESID) && x.n_per > 0;
  };
  return plain(a) && plain(b) && a.wdtype == 1 && a.K <= 2048 && b.wdtype == 0 && b.K <= 4096;
}

hipError_t launch_linear_pair(const LinearArgs& a, const LinearArgs& b, hipStream_t s) {
  if (!linear_pair_ok(a, b)) return hipErrorInvalidValue;
  const int na = gv_plan(a).blocks, nb = gv_plan(b).blocks;
  hipLaunchKernelGGL((gemv1k_pair_kernel<1, 2>), dim3(na + nb), dim3(256), 0, s, a, b, na);
  return hipGetLastError();
}

int argmax_parts_max(int n_out) {
  const int groups = ((n_out + 1) / 2 + GV_WAVES - 1) / GV_WAVES;
  const int tiles = (n_out + 15) / 16;
  return groups > tiles ? groups : tiles;
}

bool skinny_ok(int M, int K, int wdtype) { return wdtype == 1 && M >= 2 && M <= 128 && K % 64 == 0; }

int skinny_blocks(int n_out) { return (n_out + 15) / 16; }

// The skinny launch shape.  The kernels are bound by the issue of their vector loads (their
// address path stalls on the L1), not by the loads' bytes, so the shape is the one that issues the
// fewest loads on the busiest compute unit: (blocks per unit, rounded up) x (loads per wave and
// K step of a block).  Whole tiles, NT per block (grid rows of 16 input rows): NT x matrices x 2
// weight loads and 2 input loads (PACK) or 4 (two planes).  Half tiles (at most 8 rows), NH per
// block: NH x matrices weight loads and 2 input loads.  Ties go to whole tiles, then to fewer
// blocks.  Measured at the verify chunks (6 rows) against one tile per block, FlanT5-xl: W_o, the
// cross-attention projections and down (128 tiles) on one half tile a block 7.5 -> 7.0, 6.9 ->
// 6.2 and 12.7 -> 10.8 us, QKV (384 tiles) on two tiles 12.0 -> 11.5 us; LLaMA-7B shape: QKV
// (768 tiles) and gate/up (688 per matrix) on three tiles, verify 3864 -> 3686 us, where two tiles
// (the model's 12 against 8 loads) lose: 4008 us.  The LM head's argmax launch keeps four tiles.
struct SkinnyShape {
  bool half;
  int n;  // tiles or half tiles per block
};

SkinnyShape skinny_shape(int n_out, int M, int epi, bool gated) {
  const int tiles = skinny_blocks(n_out), nb = gated ? 2 : 1;
  if (epi == EPI_ARGMAX) return {false, 4};
  const bool pack = M <= 8;
  const long long cus = device_cus(), groups = pack ? 1 : (M + 15) / 16;
  SkinnyShape best = {false, 1};
  long long best_cost = -1;
  for (int nt = 1; nt <= 3; ++nt) {
    const long long blocks = (long long)((tiles + nt - 1) / nt) * groups;
    const long long cost = ((blocks + cus - 1) / cus) * (nt * nb * 2 + (pack ? 2 : 4));
    if (best_cost < 0 || cost < best_cost) { best = {false, nt}; best_cost = cost; }
  }
  // a residual epilogue on half tiles leaves a partial sum of squares per half tile (at most
  // SSQ_MAX for its consumer)
  if (pack && (epi != EPI_RESID || 2 * tiles <= SSQ_MAX)) {
    for (int nh = 1; nh <= 3; ++nh) {
      const long long blocks = (2LL * tiles + nh - 1) / nh;
      const long long cost = ((blocks + cus - 1) / cus) * (nh * nb + 2);
      if (cost < best_cost) { best = {true, nh}; best_cost = cost; }
    }
  }
  return best;
}

int skinny_ssq_parts(int n_out, int M) {
  return (skinny_shape(n_out, M, EPI_RESID, false).half ? 2 : 1) * skinny_blocks(n_out);
}

// Steps per batch of loads that the registers hold, by 16-byte weight loads per lane and step
// (wl: whole tiles NT x matrices x 2, half tiles NH x matrices) and input loads per step (il):
// with one input plane about 48 loads of 16 bytes per lane and batch (12, 8, 4 or 2 steps); the
// two-plane form (il = 4) 16 / wl steps.
constexpr int skinny_cap(int wl, int il) {
  return il == 4 ? (16 / wl > 0 ? 16 / wl : 1)
                 : (48 / (wl + il) >= 12 ? 12 : (48 / (wl + il) >= 8 ? 8 : (48 / (wl + il) >= 4 ? 4 : 2)));
}

// (only the depths the launcher can pick for each variant are instantiated)
template <bool PACK, int SK, int NT, bool G>
void launch_skinny_nt(const LinearArgs& b, bool rms, int tiles, dim3 block, hipStream_t s) {
  if constexpr (SK <= skinny_cap(NT * (G ? 2 : 1) * 2, PACK ? 2 : 4)) {
    const dim3 grid((tiles + NT - 1) / NT, (b.M + 15) / 16);
    if (rms) hipLaunchKernelGGL((gemv_mfma_kernel<G, true, NT, PACK, SK>), grid, block, 0, s, b);
    else hipLaunchKernelGGL((gemv_mfma_kernel<G, false, NT, PACK, SK>), grid, block, 0, s, b);
  }
}

template <int SK, int NH, bool G>
void launch_skinny_nh(const LinearArgs& b, bool rms, int tiles, dim3 block, hipStream_t s) {
  if constexpr (SK <= skinny_cap(NH * (G ? 2 : 1), 2)) {
    const dim3 grid((2 * tiles + NH - 1) / NH, 1);
    if (rms) hipLaunchKernelGGL((gemv_mfma_half_kernel<G, true, NH, SK>), grid, block, 0, s, b);
    else hipLaunchKernelGGL((gemv_mfma_half_kernel<G, false, NH, SK>), grid, block, 0, s, b);
  }
}

template <bool PACK, int SK>
void launch_skinny_sk(const LinearArgs& b, bool gated, bool rms, int tiles, SkinnyShape sh,
                      dim3 block, hipStream_t s) {
  if (b.epi == EPI_ARGMAX) return launch_skinny_nt<PACK, SK, 4, false>(b, rms, tiles, block, s);
  if constexpr (PACK) {
    if (sh.half) {
      switch (sh.n) {
        case 1:
          return gated ? launch_skinny_nh<SK, 1, true>(b, rms, tiles, block, s)
                       : launch_skinny_nh<SK, 1, false>(b, rms, tiles, block, s);
        case 2:
          return gated ? launch_skinny_nh<SK, 2, true>(b, rms, tiles, block, s)
                       : launch_skinny_nh<SK, 2, false>(b, rms, tiles, block, s);
        default:
          return gated ? launch_skinny_nh<SK, 3, true>(b, rms, tiles, block, s)
                       : launch_skinny_nh<SK, 3, false>(b, rms, tiles, block, s);
      }
    }
  }
  switch (sh.n) {
    case 1:
      return gated ? launch_skinny_nt<PACK, SK, 1, true>(b, rms, tiles, block, s)
                   : launch_skinny_nt<PACK, SK, 1, false>(b, rms, tiles, block, s);
    case 2:
      return gated ? launch_skinny_nt<PACK, SK, 2, true>(b, rms, tiles, block, s)
                   : launch_skinny_nt<PACK, SK, 2, false>(b, rms, tiles, block, s);
    default:
      return gated ? launch_skinny_nt<PACK, SK, 3, true>(b, rms, tiles, block, s)
                   : launch_skinny_nt<PACK, SK, 3, false>(b, rms, tiles, block, s);
  }
}

// Steps per batch: as many as the registers allow (skinny_cap), then balanced so that the wave's
// last batch is not a short one padded with clamped re-reads.  Instantiated depths: 1, 2, 4, 8,
// 10, 12 (the smallest not below the balanced depth, at most the cap).
int skinny_depth(int K, int cap) {
  const int spw = (K / 64 + SKW - 1) / SKW;
  const int batches = (spw + cap - 1) / cap;
  const int want = (spw + batches - 1) / batches;
  const int opts[6] = {1, 2, 4, 8, 10, 12};
  for (int i = 0; i < 6; ++i)
    if (opts[i] >= want && opts[i] <= cap) return opts[i];
  return cap;
}

template <bool PACK>
hipError_t launch_skinny_as(const LinearArgs& b, bool gated, bool rms, int tiles, dim3 block,
                            hipStream_t s) {
  const SkinnyShape sh = skinny_shape(gated ? b.n_per : b.n_per * b.n_mats, b.M, b.epi, gated);
  const int nb = gated ? 2 : 1;
  const int cap = sh.half ? skinny_cap(sh.n * nb, 2) : skinny_cap(sh.n * nb * 2, PACK ? 2 : 4);
  switch (skinny_depth(b.K, cap)) {
    case 1: launch_skinny_sk<PACK, 1>(b, gated, rms, tiles, sh, block, s); break;
    case 2: launch_skinny_sk<PACK, 2>(b, gated, rms, tiles, sh, block, s); break;
    case 4: launch_skinny_sk<PACK, 4>(b, gated, rms, tiles, sh, block, s); break;
    case 8: launch_skinny_sk<PACK, 8>(b, gated, rms, tiles, sh, block, s); break;
    case 10: launch_skinny_sk<PACK, 10>(b, gated, rms, tiles, sh, block, s); break;
    default: launch_skinny_sk<PACK, 12>(b, gated, rms, tiles, sh, block, s); break;
  }
  return hipGetLastError();
}

hipError_t launch_linear_skinny(const LinearArgs& a, hipStream_t s, int* n_parts) {
  const bool gated = (a.epi == EPI_GATED_GELU || a.epi == EPI_GATED_SILU);
  const int n_out = gated ? a.n_per : a.n_per * a.n_mats;
  const int tiles = skinny_blocks(n_out);
  if (!a.in_planes || a.norm == NORM_LN || a.plane_rows % 16 || a.M > a.plane_rows) return hipErrorInvalidValue;
  if (a.norm == NORM_RMS && (!a.in_ssq || a.in_nssq < 1 || a.in_nssq > SSQ_MAX)) return hipErrorInvalidValue;
  if (a.epi == EPI_QKV && (a.n_mats != 3 || (a.d_head / 2) % 8 != 0)) return hipErrorInvalidValue;
  LinearArgs b = a;
  if (b.epi == EPI_ARGMAX) b.n_parts = tiles;
  if (n_parts) *n_parts = b.n_parts;
  const bool rms = a.norm == NORM_RMS;
  const dim3 block(64 * SKW);
  if (a.M <= 8) return launch_skinny_as<true>(b, gated, rms, tiles, block, s);
  return launch_skinny_as<false>(b, gated, rms, tiles, block, s);
}

bool skinny_fold_ok(int d_model, int n_fold, int group, int M) {
  // the output projection's partial sums of squares must be those of half tiles, which the
  // chunk's other residual launches leave too
  return M >= 2 && M <= 8 && d_model % 64 == 0 && n_fold % 64 == 0 &&
         (group == 8 || group == 16 || group == 32) && n_fold % group == 0 &&
         skinny_shape(d_model, M, EPI_RESID, false).half;
}

template <int MODE, bool RMS, int SK>
void launch_fold_sk(const LinearArgs& b, int tiles, hipStream_t s) {
  hipLaunchKernelGGL((gemv_mfma_half_kernel<false, RMS, 1, SK, MODE>), dim3(2 * tiles), dim3(64 * SKW),
                     0, s, b);
}

template <int MODE, bool RMS>
void launch_fold_mode(const LinearArgs& b, int tiles, int sk, hipStream_t s) {
  switch (sk) {
    case 1: launch_fold_sk<MODE, RMS, 1>(b, tiles, s); break;
    case 2: launch_fold_sk<MODE, RMS, 2>(b, tiles, s); break;
    case 4: launch_fold_sk<MODE, RMS, 4>(b, tiles, s); break;
    case 8: launch_fold_sk<MODE, RMS, 8>(b, tiles, s); break;
    case 10: launch_fold_sk<MODE, RMS, 10>(b, tiles, s); break;
    default: launch_fold_sk<MODE, RMS, 12>(b, tiles, s); break;
  }
}

hipError_t launch_linear_skinny_fold(const LinearArgs& a, hipStream_t s) {
  const bool smx = a.norm == NORM_SOFTMAX;
  if (a.wdtype != SSD_F32 || a.n_mats != 1 || a.M < 2 || a.M > 8 || a.M > a.plane_rows ||
      a.K % 64 || a.n_per < 1)
    return hipErrorInvalidValue;
  if (smx) {
    if (a.epi != EPI_RESID || !a.in_f32 || a.in_ld % 4 ||
        (a.group != 8 && a.group != 16 && a.group != 32) || a.K % a.group)
      return hipErrorInvalidValue;
  } else if (a.norm != NORM_RMS || a.epi != EPI_STORE || !a.in_planes || !a.in_ssq ||
             a.in_nssq < 1 || a.in_nssq > SSQ_MAX) {
    return hipErrorInvalidValue;
  }
  const int tiles = skinny_blocks(a.n_per);
  // a half tile a block; 32 bytes of float32 weights and two input loads a step
  const int sk = skinny_depth(a.K, skinny_cap(2, 2));
  if (smx) launch_fold_mode<2, false>(a, tiles, sk, s);
  else launch_fold_mode<1, true>(a, tiles, sk, s);
  return hipGetLastError();
}

hipError_t launch_skinny_prep(const float* x, int ldx, int M, int K, const float* gain, bf16_t* out,
                              int ldo, int plane_rows, float* ssq, hipStream_t s) {
  if (M < 1 || M > plane_rows || K % 4) return hipErrorInvalidValue;
  hipLaunchKernelGGL(skinny_prep_kernel, dim3(M), dim3(256), 0, s, x, ldx, K, gain, out, ldo,
                     plane_rows, ssq);
  return hipGetLastError();
}

hipError_t launch_row_stats(const float* x, int ldx, int M, int K, int norm, float eps,
                            float2* stats, hipStream_t s) {
  hipLaunchKernelGGL(row_stats_kernel, dim3(M), dim3(64), 0, s, x, ldx, M, K, norm, eps, stats);
  return hipGetLastError();
}

bool linear_is_vector(const LinearArgs& a) { return !want_mfma(a); }

double linear_bytes(const LinearArgs& a) {
  const bool gated = (a.epi == EPI_GATED_GELU || a.epi == EPI_GATED_SILU);
  const double n_w = (double)a.n_per * (gated ? 2 : a.n_mats);
  const double n_out = gated ? a.n_per : n_w;
  const double welem = a.wdtype == 1 ? 2.0 : 4.0;
  double bytes = n_w * a.K * welem + (double)a.M * a.K * 4.0;
  if (a.epi == EPI_ARGMAX) bytes += a.logits ? (double)a.M * n_out * 4.0 : 0.0;
  else bytes += (double)a.M * n_out * 4.0 * (a.epi == EPI_RESID || a.epi == EPI_BIAS_RESID ? 2.0 : 1.0);
  return bytes;
}

template <bool GATED, int BN, bool RMS>
void launch_gemm2_n(const LinearArgs& a, dim3 grid, hipStream_t s) {
  constexpr int NB = GATED ? 2 : 1;
  const size_t shm = ((size_t)4 * G2M * G2KP + (size_t)2 * NB * BN * G2KP) * sizeof(bf16_t);
  static bool attr = false;
  if (!attr) {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm2_kernel<GATED, BN, RMS>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm);
    attr = true;
  }
  hipLaunchKernelGGL((gemm2_kernel<GATED, BN, RMS>), grid, dim3(256), shm, s, a);
}

template <bool GATED, int BN>
void launch_gemm2(const LinearArgs& a, dim3 grid, hipStream_t s) {
  launch_gemm2_n<GATED, BN, true>(a, grid, s);
}

template <bool GATED, int TMR, int BN>
void launch_gemm3_t(const LinearArgs& a, bool rms, hipStream_t s) {
  constexpr int NB = GATED ? 2 : 1;
  const size_t shm = ((size_t)2 * TMR * G3KP * 2 + (size_t)2 * NB * BN * G3KP) * sizeof(bf16_t);
  const int n_out = GATED ? a.n_per : a.n_per * a.n_mats;
  const dim3 grid((a.M + TMR - 1) / TMR, (n_out + BN - 1) / BN, GATED ? 1 : a.ksplit);
  if (rms) hipLaunchKernelGGL((gemm3_kernel<GATED, TMR, BN, true>), grid, dim3(256), shm, s, a);
  else hipLaunchKernelGGL((gemm3_kernel<GATED, TMR, BN, false>), grid, dim3(256), shm, s, a);
}

// Ranges of K for the tile path's residual projections: as many as keep every block of the grid
// resident at once (two 128 x 128 blocks per compute unit: 61 KB of LDS each).  At the
// LLaMA-7B shape's 608-row prefix (160 tiles over 4096 outputs) that is 3, measured faster than
// 2 or 4 (whose fourth range spills into a second round of blocks) and than the 64 x 64 tiles.
int ksplit_choice(int tiles) { return (2 * device_cus()) / tiles; }

// The plane GEMM when its buffer is there and the shape fits: RMSNorm or no norm, no argmax, K in
// whole steps, tiles that never straddle matrices.  128 x 128 tiles (gated: 128 x 64 per matrix)
// when they give at least 256 blocks, else 64 x 64.
bool try_gemm3(LinearArgs a, hipStream_t s, hipError_t* err) {
  const bool gated = (a.epi == EPI_GATED_GELU || a.epi == EPI_GATED_SILU);
  if (!a.gemm_planes || a.wdtype != 1 || a.epi == EPI_ARGMAX || a.epi == EPI_QKV) return false;
  if (a.norm != NORM_NONE && a.norm != NORM_RMS) return false;
  if (a.K % G3K || a.K > a.gemm_plane_ld || a.M > a.gemm_plane_rows || a.ldx % 4) return false;
  const int n_out = gated ? a.n_per : a.n_per * a.n_mats;
  const bool big = gated || (long long)((a.M + 127) / 128) * ((n_out + 127) / 128) >= 256;
  const int bn = gated ? 64 : (big ? 128 : 64);
  if (!gated && a.n_mats > 1 && a.n_per % bn) return false;
  const bool rms = a.norm == NORM_RMS;
  hipLaunchKernelGGL(plane_prep_kernel, dim3(a.M), dim3(256), 0, s, a.x, a.ldx, a.K,
                     rms ? a.gain : nullptr, a.eps, a.gemm_planes, a.gemm_plane_ld,
                     a.gemm_plane_rows, a.stats);
  a.in_planes = a.gemm_planes;
  a.in_ld = a.gemm_plane_ld;
  a.plane_rows = a.gemm_plane_rows;
  a.ksplit = 1;
  // residual projections with too few 128 x 128 tiles: 128 x 128 tiles over S ranges of K, then
  // the ordered sum of the S partials into y
  if (!gated && !big && a.epi == EPI_RESID && a.kpart && a.M > 128 && n_out % 4 == 0 &&
      n_out <= a.kpart_ld && a.ldy % 4 == 0 && (!a.stash || a.lds % 4 == 0)) {
    const int tiles = ((a.M + 127) / 128) * ((n_out + 127) / 128);
    const int nk = a.K / G3K;
    int S = ksplit_choice(tiles);
    if (S > a.kpart_max) S = a.kpart_max;
    if (S > 4) S = 4;
    while (S > 1 && (nk + S - 1) / S * (S - 1) >= nk) --S;  // every range holds a step
    if (S > 1) {
      a.ksplit = S;
      launch_gemm3_t<false, 128, 128>(a, rms, s);
      const int nq = a.M * (n_out / 4);
      hipLaunchKernelGGL(ksum_kernel, dim3((nq + 255) / 256), dim3(256), 0, s, a, n_out);
      *err = hipGetLastError();
      return true;
    }
  }
  if (gated) launch_gemm3_t<true, 128, 64>(a, rms, s);
  else if (big) launch_gemm3_t<false, 128, 128>(a, rms, s);
  else launch_gemm3_t<false, 64, 64>(a, rms, s);
  *err = hipGetLastError();
  return true;
}

hipError_t launch_linear(LinearArgs a, hipStream_t s, int* n_parts, LaunchTiming* timing) {
  if (a.M <= 0) return hipSuccess;
  // the softmax input transform exists on the one-row register path only
  if (a.norm == NORM_SOFTMAX &&
      (a.M != 1 || a.K > 6144 || (a.group != 8 && a.group != 16 && a.group != 32 && a.group != 64) ||
       a.K % a.group))
    return hipErrorInvalidValue;
  const bool gated = (a.epi == EPI_GATED_GELU || a.epi == EPI_GATED_SILU);
  const int n_out = gated ? a.n_per : a.n_per * a.n_mats;
  if (want_mfma(a)) {
    a.use_mfma = 1;
    if (a.epi == EPI_ARGMAX) a.n_parts = (n_out + TN - 1) / TN;
    if (n_parts) *n_parts = a.n_parts;
    hipError_t e3 = hipSuccess;
    if (try_gemm3(a, s, &e3)) return e3;
    if (a.norm != NORM_NONE) {
      hipError_t e = launch_row_stats(a.x, a.ldx, a.M, a.K, a.norm, a.eps, a.stats, s);
      if (e != hipSuccess) return e;
    }
    // long row blocks with a normalised input (QKV, cross query, gate/up): 128-row tiles with
    // double buffering (measured faster than the 64x64 tiles there; the residual projections keep
    // the 64x64 tiles, whose larger grids hide the memory latency better)
    if (a.epi != EPI_ARGMAX && a.norm == NORM_RMS && a.M > 64 && a.K % G2K == 0) {
      const int bn = gated ? 64 : 128;
      if (a.n_mats == 1 || gated || a.n_per % bn == 0) {
        dim3 grid((a.M + G2M - 1) / G2M, (n_out + bn - 1) / bn);
        if (gated) launch_gemm2<true, 64>(a, grid, s);
        else launch_gemm2<false, 128>(a, grid, s);
        return hipGetLastError();
      }
    }
    dim3 grid((n_out + TN - 1) / TN, (a.M + TM - 1) / TM);
    if (gated) hipLaunchKernelGGL((gemm_kernel<true>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((gemm_kernel<false>), grid, dim3(256), 0, s, a);
    return hipGetLastError();
  }
  a.use_mfma = 0;
  if (a.epi == EPI_ARGMAX) a.n_parts = gv_plan(a).blocks;
  if (n_parts) *n_parts = a.n_parts;
  if (use_gemv1k(a)) return launch_gemv1k_any(a, s, timing);
  return a.wdtype == 1 ? launch_gemv_t<bf16_t>(a, s, timing) : launch_gemv_t<float>(a, s, timing);
}

}  // namespace ssd
