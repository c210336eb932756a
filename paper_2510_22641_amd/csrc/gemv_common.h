// Device helpers of the weight-streaming GEMV kernels (linear.hip): row-pair
// addressing of the concatenated / gated matrices, the QKV epilogue (rotary and the paged KV
// store), and the fused epilogues of the vector path for up to MB input rows.
#pragma once

#include "device.h"
#include "kernels.h"

#include <climits>

namespace ssd {

namespace {

constexpr int GV_WAVES = 4;
constexpr int GV_LDS_FLOATS = 36864;    // 144 KB of staged input rows per block (160 KB LDS)

__device__ __forceinline__ float apply_epi_act(int epi, float g, float u) {
  return (epi == EPI_GATED_GELU ? gelu_tanh(g) : silu(g)) * u;
}

// Weight rows of one wave's current row pair: two consecutive rows of one of the concatenated
// matrices, or the (gate, up) rows of one FFN feature.
template <typename WT>
struct RowPair {
  const WT* w0;
  const WT* w1;
  int n0, n1;  // output columns (virtual rows)
  bool ok0, ok1;
};

template <typename WT>
__device__ __forceinline__ RowPair<WT> row_pair(const LinearArgs& a, bool gated, int n_total, int pr) {
  RowPair<WT> r;
  const int K = a.K;
  if (gated) {
    r.ok0 = r.ok1 = pr < a.n_per;
    const int q = r.ok0 ? pr : 0;
    r.n0 = r.n1 = pr;
    r.w0 = reinterpret_cast<const WT*>(a.w[0]) + (size_t)q * K;
    r.w1 = reinterpret_cast<const WT*>(a.w[1]) + (size_t)q * K;
    return r;
  }
  if (a.epi == EPI_QKV) {
    // the pair (i, i + d_head/2) of one head of one matrix: the rotary pair
    const int hd2 = a.n_per >> 1, half = a.d_head >> 1;
    r.ok0 = r.ok1 = pr < 3 * hd2;
    const int q = r.ok0 ? pr : 0;
    const int mat = q >= hd2 ? (q >= 2 * hd2 ? 2 : 1) : 0;
    const int loc = q - mat * hd2;
    const int h = loc / half, i = loc - h * half;
    const int c0 = h * a.d_head + i;
    r.n0 = mat * a.n_per + c0;
    r.n1 = r.n0 + half;
    // select among the three matrix pointers (an indexed a.w[mat] would be fetched from the
    // argument buffer by a vector load, making the weight loads wait for the inputs)
    const void* base = mat == 0 ? a.w[0] : (mat == 1 ? a.w[1] : a.w[2]);
    r.w0 = reinterpret_cast<const WT*>(base) + (size_t)c0 * K;
    r.w1 = r.w0 + (size_t)half * K;
    return r;
  }
  r.n0 = 2 * pr;
  r.n1 = 2 * pr + 1;
  r.ok0 = r.n0 < n_total;
  r.ok1 = r.n1 < n_total;
  int v0 = r.ok0 ? r.n0 : 0, v1 = r.ok1 ? r.n1 : v0;
  // locate each virtual row in its matrix without a division (at most three matrices)
  const void* b0 = a.w[0];
  if (v0 >= a.n_per) { v0 -= a.n_per; b0 = a.w[1]; if (v0 >= a.n_per) { v0 -= a.n_per; b0 = a.w[2]; } }
  const void* b1 = a.w[0];
  if (v1 >= a.n_per) { v1 -= a.n_per; b1 = a.w[1]; if (v1 >= a.n_per) { v1 -= a.n_per; b1 = a.w[2]; } }
  r.w0 = reinterpret_cast<const WT*>(b0) + (size_t)v0 * K;
  r.w1 = reinterpret_cast<const WT*>(b1) + (size_t)v1 * K;
  return r;
}

// EPI_QKV epilogue of one rotary pair (columns c0 and c0 + d_head/2 of q, k or v) for the
// block's input rows: rotate q and k by the row's position, then store q to y and k / v into
// their page.  A position past the cache or an unmapped page sets a status bit and skips the KV
// store.
template <typename KT>
__device__ __forceinline__ void store_kv_pair(const LinearArgs& a, int page, int slot, int h, int i,
                                              int half, bool is_v, float e0, float e1) {
  KT* base = reinterpret_cast<KT*>(is_v ? a.kv.v : a.kv.k) +
             (((size_t)page * a.n_heads + h) * a.kv.page_size + slot) * a.d_head;
  store_elem(base + i, e0);
  store_elem(base + i + half, e1);
}

// Where the pair (c0, c0 + d_head/2) of input row `row` goes: the row's position, its rotary
// factors and the page entry that holds it.  Split in two so that a kernel can request the
// sequence length before its weights and the dependent page-table and rotary entries right after
// them (every load is clamped to a valid address; validity is decided at the store).
struct QkvPre {
  int pos, page;
  float cs, sn;
};

__device__ __forceinline__ int qkv_pos(const LinearArgs& a, int row) {
  const int b = row / a.C, j = row - b * a.C;
  return a.kv.seq_len[b] + a.kv.pos_off + j;
}

__device__ __forceinline__ QkvPre qkv_pre(const LinearArgs& a, int mat, int c0, int row, int pos) {
  QkvPre p;
  p.pos = pos;
  p.cs = 1.f;
  p.sn = 0.f;
  const int half = a.d_head >> 1;
  const int i = c0 % a.d_head;
  if (mat < 2 && a.rope_cos) {
    const int tp = pos < 0 ? 0 : (pos >= a.max_seq ? a.max_seq - 1 : pos);
    p.cs = a.rope_cos[(size_t)tp * half + i];
    p.sn = a.rope_sin[(size_t)tp * half + i];
  }
  const int b = row / a.C;
  const int pg_i = pos >= 0 ? pos / a.kv.page_size : 0;
  p.page = a.kv.page_table[(size_t)b * a.kv.max_pages + min(pg_i, a.kv.max_pages - 1)];
  return p;
}

// Rotary (q, k) and the store of one pair of input row `row`: columns c0 and c0 + d_head/2 of
// matrix mat (0 = q -> y, 1 = k, 2 = v -> the row's page).  A position past the cache or an
// unmapped page sets a status bit and skips the KV store.
__device__ __forceinline__ void qkv_store_pre(const LinearArgs& a, int mat, int c0, int row,
                                              const QkvPre& p, float e0, float e1) {
  const int half = a.d_head >> 1;
  const int h = c0 / a.d_head, i = c0 - h * a.d_head;
  if (mat < 2 && a.rope_cos) {
    const float r0 = e0 * p.cs - e1 * p.sn, r1 = e1 * p.cs + e0 * p.sn;
    e0 = r0;
    e1 = r1;
  }
  if (mat == 0) {
    a.y[(size_t)row * a.ldy + c0] = e0;
    a.y[(size_t)row * a.ldy + c0 + half] = e1;
    return;
  }
  const int pos = p.pos;
  if (pos < 0 || pos >= a.max_seq || pos / a.kv.page_size >= a.kv.max_pages) {
    atomicOr(a.status, SSD_DEV_CAPACITY);
    return;
  }
  if (p.page < 0 || p.page >= a.kv.n_pages) {
    atomicOr(a.status, SSD_DEV_BAD_PAGE);
    return;
  }
  const int slot = pos % a.kv.page_size;
  if (a.kvdtype == 1) store_kv_pair<bf16_t>(a, p.page, slot, h, i, half, mat == 2, e0, e1);
  else store_kv_pair<float>(a, p.page, slot, h, i, half, mat == 2, e0, e1);
}

__device__ __forceinline__ void qkv_store_pair(const LinearArgs& a, int mat, int c0, int row,
                                               float e0, float e1) {
  qkv_store_pre(a, mat, c0, row, qkv_pre(a, mat, c0, row, qkv_pos(a, row)), e0, e1);
}

template <int MB>
__device__ __forceinline__ void qkv_epilogue(const LinearArgs& a, int n0, const float (&acc)[2][MB],
                                             int m0, int mrows) {
  const int HD = a.n_per;
  const int mat = n0 >= HD ? (n0 >= 2 * HD ? 2 : 1) : 0;
#pragma unroll
  for (int m = 0; m < MB; ++m) {
    if (m >= mrows) break;
    qkv_store_pair(a, mat, n0 - mat * HD, m0 + m, acc[0][m], acc[1][m]);
  }
}

// Unconditional loads (a tail piece past K re-reads the row's last 8 elements and is skipped by
// fma_pieces): a conditional zero fill would make the compiler drain every pending load first.
template <typename WT, int GV_KP>
__device__ __forceinline__ void load_pieces(Vec8<WT> (&buf)[2][GV_KP], const RowPair<WT>& r, int e0,
                                            int K, int lane) {
#pragma unroll
  for (int p = 0; p < GV_KP; ++p) {
    const int e = min(e0 + p * 512 + lane * 8, K - 8);
    buf[0][p].load(r.w0 + e);
    buf[1][p].load(r.w1 + e);
  }
}

// LDS layout of the staged input rows: element k of row m sits in plane (k / 4) % 2 at
// m * ldxs + (k / 8) * 4 + k % 4 (plane 1 starts ldxs / 2 floats later), so that the two 16-byte
// reads of a lane's 8 consecutive elements are each contiguous across the wave (no bank conflicts).
__device__ __forceinline__ int xs_off(int k, int ldxs) {
  return ((k >> 3) << 2) + (k & 3) + ((k >> 2) & 1) * (ldxs >> 1);
}

template <typename WT, int MB, int GV_KP>
__device__ __forceinline__ void fma_pieces(const Vec8<WT> (&buf)[2][GV_KP], const float* xs, int ldxs,
                                           int e0, int K, int lane, float (&acc)[2][MB]) {
#pragma unroll
  for (int p = 0; p < GV_KP; ++p) {
    const int e = e0 + p * 512 + lane * 8;
    if (e < K) {
      float w0[8], w1[8];
      buf[0][p].to_f32(w0);
      buf[1][p].to_f32(w1);
      const int o = e >> 1;  // (e / 8) * 4
#pragma unroll
      for (int m = 0; m < MB; ++m) {
        const float4 xa = *reinterpret_cast<const float4*>(xs + m * ldxs + o);
        const float4 xb = *reinterpret_cast<const float4*>(xs + m * ldxs + (ldxs >> 1) + o);
        float t0 = acc[0][m], t1 = acc[1][m];
        t0 = fmaf(w0[0], xa.x, t0); t1 = fmaf(w1[0], xa.x, t1);
        t0 = fmaf(w0[1], xa.y, t0); t1 = fmaf(w1[1], xa.y, t1);
        t0 = fmaf(w0[2], xa.z, t0); t1 = fmaf(w1[2], xa.z, t1);
        t0 = fmaf(w0[3], xa.w, t0); t1 = fmaf(w1[3], xa.w, t1);
        t0 = fmaf(w0[4], xb.x, t0); t1 = fmaf(w1[4], xb.x, t1);
        t0 = fmaf(w0[5], xb.y, t0); t1 = fmaf(w1[5], xb.y, t1);
        t0 = fmaf(w0[6], xb.z, t0); t1 = fmaf(w1[6], xb.z, t1);
        t0 = fmaf(w0[7], xb.w, t0); t1 = fmaf(w1[7], xb.w, t1);
        acc[0][m] = t0; acc[1][m] = t1;
      }
    }
  }
}

// Epilogue of the vector GEMV for the block's input rows m0 .. m0 + mrows - 1: acc holds this
// wave's two outputs per row (already scaled by 1/rms when folded), yold the residual values
// lane 0 read before the weights.  Argmax partials are merged over the block's waves (one
// barrier; every thread of the block must call this).
template <typename WT, int MB>
__device__ __forceinline__ void gemv_finish(const LinearArgs& a, const RowPair<WT>& r,
                                            const float (&acc)[2][MB], const float (&yold)[2][MB],
                                            bool live, bool gated, bool argmax, int m0, int mrows,
                                            int tid, int lane, int wave, float (&rv)[GV_WAVES][MB],
                                            int (&ri)[GV_WAVES][MB], const QkvPre& pre = {},
                                            bool use_pre = false) {
  float best_v[MB];
  int best_i[MB];
#pragma unroll
  for (int m = 0; m < MB; ++m) {
    best_v[m] = -INFINITY;
    best_i[m] = INT_MAX;
  }
  if (argmax) {
    if (live) {
#pragma unroll
      for (int m = 0; m < MB; ++m) {
        if (r.ok0) argmax_merge(best_v[m], best_i[m], acc[0][m], r.n0);
        if (r.ok1) argmax_merge(best_v[m], best_i[m], acc[1][m], r.n1);
        if (a.logits && lane == 0 && m < mrows) {
          float* lp = a.logits + (size_t)(m0 + m) * a.ldl;
          if (r.ok0) lp[r.n0] = acc[0][m];
          if (r.ok1) lp[r.n1] = acc[1][m];
        }
      }
    }
  } else if (lane == 0 && live && a.epi == EPI_QKV) {
    if (use_pre) {
      const int HD = a.n_per, mat = r.n0 >= HD ? (r.n0 >= 2 * HD ? 2 : 1) : 0;
      qkv_store_pre(a, mat, r.n0 - mat * HD, m0, pre, acc[0][0], acc[1][0]);
    } else {
      qkv_epilogue<MB>(a, r.n0, acc, m0, mrows);
    }
  } else if (lane == 0 && live) {
#pragma unroll
    for (int m = 0; m < MB; ++m) {
      if (m >= mrows) break;
      const size_t row = (size_t)(m0 + m);
      if (gated) {
        if (r.ok0) a.y[row * a.ldy + r.n0] = apply_epi_act(a.epi, acc[0][m], acc[1][m]);
        continue;
      }
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        const bool ok = s ? r.ok1 : r.ok0;
        if (!ok) continue;
        const int n = s ? r.n1 : r.n0;
        const float v = acc[s][m];
        float* yp = a.y + row * a.ldy + n;
        if (a.epi == EPI_STORE) {
          *yp = v;
        } else if (a.epi == EPI_RESID) {
          const float t = yold[s][m] + v;
          *yp = t;
          if (a.stash) a.stash[row * a.lds + n] = t;
        } else if (a.epi == EPI_BIAS_GELU) {
          *yp = gelu_tanh(v + a.bias[n]);
        } else if (a.epi == EPI_BIAS_RESID) {
          *yp = yold[s][m] + (v + (a.bias ? a.bias[n] : 0.f));
        }
      }
    }
  }

  if (!argmax) return;
  // block's best per row -> one partial per (row, block); launch_argmax_final reduces them
  if (lane == 0) {
#pragma unroll
    for (int m = 0; m < MB; ++m) { rv[wave][m] = best_v[m]; ri[wave][m] = best_i[m]; }
  }
  __syncthreads();
  if (tid < mrows) {
    const int m = tid;
    float v = rv[0][m];
    int i = ri[0][m];
    for (int ww = 1; ww < GV_WAVES; ++ww) argmax_merge(v, i, rv[ww][m], ri[ww][m]);
    a.part_val[(size_t)(m0 + m) * a.n_parts + blockIdx.x] = v;
    a.part_idx[(size_t)(m0 + m) * a.n_parts + blockIdx.x] = i;
  }
}

}  // namespace

}  // namespace ssd
