// Softmax attention of a block of query rows of one head.
//
// Self-attention: query row j of sequence b sits at position p = seq_len[b] + pos_off + j and
// attends keys 0..p of the paged cache (causal inside a verify chunk or a prefill block), with the
// T5 relative-position bias bias[h][p - i] added (no scaling; T5 folds it into the weights) or,
// for LLaMA, scaled by 1/sqrt(dh) with q and k already rotated.  Cross-attention (T5): all n_keys
// visual keys, no mask, no bias, no scale.
//
// One block per (head, sequence, 8 query rows): scores for the 8 rows over all keys go to LDS,
// one wave per row normalises them, and each wave accumulates P.V for two rows with one lane per
// head dimension (coalesced 128-byte value rows).  Bound: bytes of K and V read (HBM/L2).
#include "device.h"
#include "kernels.h"

namespace ssd {

namespace {

constexpr int QB = 8;

template <typename KT, int DH>
__device__ __forceinline__ const KT* key_row(const AttnArgs& a, const KT* base, int b, int h, int i,
                                             bool& ok) {
  if (a.cross) {
    ok = true;
    return base + ((size_t)(b * a.H + h) * a.n_keys + i) * DH;
  }
  const int pg_i = i / a.kv.page_size;
  int page = -1;
  if (pg_i < a.kv.max_pages) page = a.kv.page_table[(size_t)b * a.kv.max_pages + pg_i];
  ok = page >= 0 && page < a.kv.n_pages;
  if (!ok) page = 0;
  const int slot = i - pg_i * a.kv.page_size;
  return base + (((size_t)page * a.H + h) * a.kv.page_size + slot) * DH;
}

template <typename KT, int DH>
__global__ __launch_bounds__(256) void attn_kernel(const AttnArgs a, const int s_stride) {
  extern __shared__ float S[];  // [QB][s_stride]
  __shared__ float qs[QB][DH];
  __shared__ float inv_sum[QB];

  const int h = blockIdx.x, b = blockIdx.y, j0 = blockIdx.z * QB;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nq = min(QB, a.C - j0);
  const int HD = a.H * DH;
  const int base = a.cross ? 0 : a.kv.seq_len[b] + a.kv.pos_off;
  int nk = a.cross ? a.n_keys : base + j0 + nq;
  if (nk > s_stride) {
    if (tid == 0) atomicOr(a.status, SSD_DEV_CAPACITY);
    nk = s_stride;
  }
  const KT* Kb = reinterpret_cast<const KT*>(a.cross ? a.xk : a.kv.k);
  const KT* Vb = reinterpret_cast<const KT*>(a.cross ? a.xv : a.kv.v);

  for (int idx = tid; idx < QB * DH; idx += 256) {
    const int jq = idx / DH, d = idx - jq * DH;
    qs[jq][d] = jq < nq ? a.q[(size_t)(b * a.C + j0 + jq) * HD + h * DH + d] * a.scale : 0.f;
  }
  __syncthreads();

  // scores
  for (int i = tid; i < nk; i += 256) {
    bool ok;
    const KT* kp = key_row<KT, DH>(a, Kb, b, h, i, ok);
    float dots[QB];
#pragma unroll
    for (int jq = 0; jq < QB; ++jq) dots[jq] = 0.f;
    if (ok) {
#pragma unroll
      for (int dc = 0; dc < DH; dc += 8) {
        Vec8<KT> kv;
        kv.load(kp + dc);
        float kf[8];
        kv.to_f32(kf);
#pragma unroll
        for (int jq = 0; jq < QB; ++jq) {
          float t = dots[jq];
#pragma unroll
          for (int e = 0; e < 8; ++e) t = fmaf(qs[jq][dc + e], kf[e], t);
          dots[jq] = t;
        }
      }
    }
#pragma unroll
    for (int jq = 0; jq < QB; ++jq) {
      float s = dots[jq];
      if (!ok || jq >= nq) {
        s = -INFINITY;
      } else if (!a.cross) {
        const int p = base + j0 + jq;
        if (i > p) s = -INFINITY;
        else if (a.bias && p - i < a.max_seq) s += a.bias[(size_t)h * a.max_seq + (p - i)];
      }
      S[jq * s_stride + i] = s;
    }
  }
  __syncthreads();

  // softmax, one wave per row
  for (int jq = wave; jq < nq; jq += 4) {
    float* row = S + jq * s_stride;
    float m = -INFINITY;
    for (int i = lane; i < nk; i += 64) m = fmaxf(m, row[i]);
    m = wave_max(m);
    float sum = 0.f;
    for (int i = lane; i < nk; i += 64) {
      const float e = (m == -INFINITY || row[i] == -INFINITY) ? 0.f : expf(row[i] - m);
      row[i] = e;
      sum += e;
    }
    sum = wave_sum(sum);
    if (lane == 0) inv_sum[jq] = sum > 0.f ? 1.0f / sum : 0.f;
  }
  __syncthreads();

  // P . V: wave w handles rows w and w + 4, lane handles dims lane + 64 t
  constexpr int DT = DH / 64;
  float acc[2][DT];
#pragma unroll
  for (int r = 0; r < 2; ++r)
#pragma unroll
    for (int t = 0; t < DT; ++t) acc[r][t] = 0.f;
  const int r0 = wave, r1 = wave + 4;
  const float* P0 = S + r0 * s_stride;
  const float* P1 = S + r1 * s_stride;
  const bool has0 = r0 < nq, has1 = r1 < nq;
  int i = 0;
  for (; i + 4 <= nk; i += 4) {
    float vv[4][DT];
    bool okk[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const KT* vp = key_row<KT, DH>(a, Vb, b, h, i + u, okk[u]);
#pragma unroll
      for (int t = 0; t < DT; ++t) vv[u][t] = okk[u] ? load_elem(vp + lane + 64 * t) : 0.f;
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const float p0 = has0 ? P0[i + u] : 0.f;
      const float p1 = has1 ? P1[i + u] : 0.f;
#pragma unroll
      for (int t = 0; t < DT; ++t) {
        acc[0][t] = fmaf(p0, vv[u][t], acc[0][t]);
        acc[1][t] = fmaf(p1, vv[u][t], acc[1][t]);
      }
    }
  }
  for (; i < nk; ++i) {
    bool ok;
    const KT* vp = key_row<KT, DH>(a, Vb, b, h, i, ok);
    const float p0 = has0 ? P0[i] : 0.f;
    const float p1 = has1 ? P1[i] : 0.f;
#pragma unroll
    for (int t = 0; t < DT; ++t) {
      const float v = ok ? load_elem(vp + lane + 64 * t) : 0.f;
      acc[0][t] = fmaf(p0, v, acc[0][t]);
      acc[1][t] = fmaf(p1, v, acc[1][t]);
    }
  }
  if (has0) {
    const float s = inv_sum[r0];
    float* o = a.out + (size_t)(b * a.C + j0 + r0) * HD + h * DH;
#pragma unroll
    for (int t = 0; t < DT; ++t) o[lane + 64 * t] = acc[0][t] * s;
  }
  if (has1) {
    const float s = inv_sum[r1];
    float* o = a.out + (size_t)(b * a.C + j0 + r1) * HD + h * DH;
#pragma unroll
    for (int t = 0; t < DT; ++t) o[lane + 64 * t] = acc[1][t] * s;
  }
}

template <typename KT>
hipError_t launch_attn_t(const AttnArgs& a, hipStream_t s) {
  const int nk_max = a.cross ? a.n_keys : a.max_seq;
  const int s_stride = (nk_max + 63) & ~63;
  dim3 grid(a.H, a.B, (a.C + QB - 1) / QB);
  const size_t shm = (size_t)QB * s_stride * sizeof(float);
  if (a.dh == 64) hipLaunchKernelGGL((attn_kernel<KT, 64>), grid, dim3(256), shm, s, a, s_stride);
  else hipLaunchKernelGGL((attn_kernel<KT, 128>), grid, dim3(256), shm, s, a, s_stride);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention(const AttnArgs& a, hipStream_t s) {
  if (a.B <= 0 || a.C <= 0) return hipSuccess;
  return a.kvdtype == 1 ? launch_attn_t<bf16_t>(a, s) : launch_attn_t<float>(a, s);
}

}  // namespace ssd
