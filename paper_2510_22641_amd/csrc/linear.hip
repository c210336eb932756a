// Linear layers y = epilogue(W . norm(x)) for the decoder, the imitation network and the LM head.
//
// Two paths:
//  * gemv_kernel — weight streaming for few rows (M <= 8: the batch-1..8 draft steps and the
//    batch-1 verify chunk).  Each wave owns two output features and reads their weight rows with
//    16-byte loads (8 bf16 / 4+4 f32 per lane, 512 elements per wave per step), the first batch of
//    loads issued before the block normalises its input rows into LDS; fp32 accumulation, wave
//    reduction, fused epilogue.  Bound: HBM bytes of W.
//  * gemm_kernel — 64x64x64 tiles on v_mfma_f32_16x16x32_bf16 with LDS staging, for larger M
//    (prefill, batch-8 verify).  The fp32 inputs are normalised and rounded to bf16 while they are
//    staged.
#include "device.h"
#include "kernels.h"

#include <climits>

namespace ssd {

namespace {

constexpr int GV_WAVES = 4;
constexpr int GV_LDS_FLOATS = 12288;  // 48 KB of normalised inputs per block

// 512-element steps per prefetch batch: fewer when many rows keep many accumulators live
template <int MB> struct GvU { static constexpr int value = MB >= 8 ? 2 : 4; };

__device__ __forceinline__ float apply_epi_act(int epi, float g, float u) {
  return (epi == EPI_GATED_GELU ? gelu_tanh(g) : silu(g)) * u;
}

template <typename WT, int GV_U>
__device__ __forceinline__ void load_batch(Vec8<WT> (&buf)[2][GV_U], const WT* const (&wr)[2],
                                           int it0, int n_it, int K, int lane) {
#pragma unroll
  for (int s = 0; s < 2; ++s) {
#pragma unroll
    for (int u = 0; u < GV_U; ++u) {
      const int it = it0 + u;
      const int e = it * 512 + lane * 8;
      if (it < n_it && e < K) buf[s][u].load(wr[s] + e);
      else buf[s][u].zero();
    }
  }
}

template <typename WT, int MB>
__global__ __launch_bounds__(256) void gemv_kernel(const LinearArgs a, const int kc) {
  constexpr int GV_U = GvU<MB>::value;
  extern __shared__ float xs[];  // [MB][kc]
  __shared__ float2 st[MB];
  __shared__ float rv[GV_WAVES][MB];
  __shared__ int ri[GV_WAVES][MB];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int m0 = blockIdx.y * MB;
  const int mrows = min(MB, a.M - m0);
  const int K = a.K;
  const bool gated = (a.epi == EPI_GATED_GELU || a.epi == EPI_GATED_SILU);
  const int n_total = gated ? a.n_per : a.n_per * a.n_mats;
  const int gw = blockIdx.x * GV_WAVES + wave;

  const WT* wr[2];
  int vrow[2];
  bool ok[2];
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    if (gated) {
      ok[s] = gw < a.n_per;
      vrow[s] = gw;
      wr[s] = reinterpret_cast<const WT*>(a.w[s]) + (size_t)(ok[s] ? gw : 0) * K;
    } else {
      const int v = 2 * gw + s;
      ok[s] = v < n_total;
      vrow[s] = v;
      const int vv = ok[s] ? v : 0;
      const int mat = vv / a.n_per;
      const int r = vv - mat * a.n_per;
      const void* base = mat == 0 ? a.w[0] : (mat == 1 ? a.w[1] : a.w[2]);
      wr[s] = reinterpret_cast<const WT*>(base) + (size_t)r * K;
    }
  }

  const int n_it = (K + 511) >> 9;
  Vec8<WT> cur[2][GV_U];
  load_batch<WT, GV_U>(cur, wr, 0, n_it, K, lane);  // weights do not depend on x: start streaming now

  // row statistics of the inputs
  if (a.norm != NORM_NONE) {
    for (int m = wave; m < mrows; m += GV_WAVES) {
      const float* xr = a.x + (size_t)(m0 + m) * a.ldx;
      float mean = 0.f;
      if (a.norm == NORM_LN) {
        float s1 = 0.f;
        for (int k = lane * 4; k < K; k += 256) {
          const float4 v = *reinterpret_cast<const float4*>(xr + k);
          s1 += (v.x + v.y) + (v.z + v.w);
        }
        mean = wave_sum(s1) / (float)K;
      }
      float s2 = 0.f;
      for (int k = lane * 4; k < K; k += 256) {
        const float4 v = *reinterpret_cast<const float4*>(xr + k);
        const float a0 = v.x - mean, a1 = v.y - mean, a2 = v.z - mean, a3 = v.w - mean;
        s2 += (a0 * a0 + a1 * a1) + (a2 * a2 + a3 * a3);
      }
      s2 = wave_sum(s2);
      if (lane == 0) st[m] = make_float2(mean, 1.0f / sqrtf(s2 / (float)K + a.eps));
    }
  }

  float acc[2][MB];
#pragma unroll
  for (int s = 0; s < 2; ++s)
#pragma unroll
    for (int m = 0; m < MB; ++m) acc[s][m] = 0.f;

  for (int kc0 = 0; kc0 < K; kc0 += kc) {
    __syncthreads();
    const int kl = min(kc, K - kc0);
    for (int idx = threadIdx.x * 4; idx < MB * kc; idx += 256 * 4) {
      const int m = idx / kc, k = idx - m * kc;
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
      if (m < mrows && k < kl) {
        v = *reinterpret_cast<const float4*>(a.x + (size_t)(m0 + m) * a.ldx + kc0 + k);
        if (a.norm != NORM_NONE) {
          const float2 s = st[m];
          const float4 g = *reinterpret_cast<const float4*>(a.gain + kc0 + k);
          v.x = (v.x - s.x) * s.y * g.x;
          v.y = (v.y - s.x) * s.y * g.y;
          v.z = (v.z - s.x) * s.y * g.z;
          v.w = (v.w - s.x) * s.y * g.w;
          if (a.norm == NORM_LN) {
            const float4 b = *reinterpret_cast<const float4*>(a.shift + kc0 + k);
            v.x += b.x; v.y += b.y; v.z += b.z; v.w += b.w;
          }
        }
      }
      *reinterpret_cast<float4*>(xs + idx) = v;
    }
    __syncthreads();

    const int it_end = min(n_it, (kc0 + kc + 511) >> 9);
    for (int it0 = kc0 >> 9; it0 < it_end; it0 += GV_U) {
      Vec8<WT> nxt[2][GV_U];
      const bool more = it0 + GV_U < n_it;
      if (more) load_batch<WT, GV_U>(nxt, wr, it0 + GV_U, n_it, K, lane);
#pragma unroll
      for (int u = 0; u < GV_U; ++u) {
        const int it = it0 + u;
        const int e = it * 512 + lane * 8;
        if (it < it_end && e < K) {
          const int el = e - kc0;
          float w0[8], w1[8];
          cur[0][u].to_f32(w0);
          cur[1][u].to_f32(w1);
#pragma unroll
          for (int m = 0; m < MB; ++m) {
            const float4 xa = *reinterpret_cast<const float4*>(xs + m * kc + el);
            const float4 xb = *reinterpret_cast<const float4*>(xs + m * kc + el + 4);
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
      if (more) {
#pragma unroll
        for (int s = 0; s < 2; ++s)
#pragma unroll
          for (int u = 0; u < GV_U; ++u) cur[s][u] = nxt[s][u];
      }
    }
  }

#pragma unroll
  for (int s = 0; s < 2; ++s)
#pragma unroll
    for (int m = 0; m < MB; ++m) acc[s][m] = wave_sum(acc[s][m]);

  if (a.epi == EPI_ARGMAX) {
#pragma unroll
    for (int m = 0; m < MB; ++m) {
      float v = -INFINITY;
      int i = INT_MAX;
#pragma unroll
      for (int s = 0; s < 2; ++s)
        if (ok[s]) argmax_merge(v, i, acc[s][m], vrow[s]);
      if (lane == 0) {
        rv[wave][m] = v;
        ri[wave][m] = i;
        if (a.logits && m < mrows) {
#pragma unroll
          for (int s = 0; s < 2; ++s)
            if (ok[s]) a.logits[(size_t)(m0 + m) * a.ldl + vrow[s]] = acc[s][m];
        }
      }
    }
    __syncthreads();
    if ((int)threadIdx.x < mrows) {
      const int m = threadIdx.x;
      float v = rv[0][m];
      int i = ri[0][m];
      for (int w = 1; w < GV_WAVES; ++w) argmax_merge(v, i, rv[w][m], ri[w][m]);
      a.part_val[(size_t)(m0 + m) * a.n_parts + blockIdx.x] = v;
      a.part_idx[(size_t)(m0 + m) * a.n_parts + blockIdx.x] = i;
    }
    return;
  }

  if (lane != 0) return;
#pragma unroll
  for (int m = 0; m < MB; ++m) {
    if (m >= mrows) break;
    const size_t row = (size_t)(m0 + m);
    if (gated) {
      if (ok[0]) a.y[row * a.ldy + vrow[0]] = apply_epi_act(a.epi, acc[0][m], acc[1][m]);
      continue;
    }
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      if (!ok[s]) continue;
      const int n = vrow[s];
      const float v = acc[s][m];
      float* yp = a.y + row * a.ldy + n;
      switch (a.epi) {
        case EPI_STORE: *yp = v; break;
        case EPI_RESID: {
          const float t = *yp + v;
          *yp = t;
          if (a.stash) a.stash[row * a.lds + n] = t;
          break;
        }
        case EPI_BIAS_GELU: *yp = gelu_tanh(v + a.bias[n]); break;
        case EPI_BIAS_RESID: *yp = (a.resid ? a.resid[row * a.ldr + n] : 0.f) + (v + a.bias[n]); break;
        default: break;
      }
    }
  }
}

// ---------------------------------------------------------------------------------------------
// MFMA tile path
constexpr int TM = 64, TN = 64, TK = 64, TKP = TK + 8;

template <bool GATED>
__global__ __launch_bounds__(256) void gemm_kernel(const LinearArgs a) {
  constexpr int NB = GATED ? 2 : 1;
  __shared__ __attribute__((aligned(16))) bf16_t As[TM][TKP];
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
    const uint4 pa0 = pack_bf16x8(f), pa1 = pack_bf16x8(f + 8);
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
    *reinterpret_cast<uint4*>(&As[lr][lk]) = pa0;
    *reinterpret_cast<uint4*>(&As[lr][lk + 8]) = pa1;
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      *reinterpret_cast<uint4*>(&Bs[b][lr][lk]) = pb[b][0];
      *reinterpret_cast<uint4*>(&Bs[b][lr][lk + 8]) = pb[b][1];
    }
    __syncthreads();
#pragma unroll
    for (int ks = 0; ks < TK; ks += 32) {
      const int kk = ks + (lane >> 4) * 8;
      bf16x8_t af[2], bfr[NB][2];
#pragma unroll
      for (int i = 0; i < 2; ++i)
        af[i] = *reinterpret_cast<const bf16x8_t*>(&As[wm + 16 * i + (lane & 15)][kk]);
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
          for (int j = 0; j < 2; ++j)
            acc[b][i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[b][j], acc[b][i][j], 0, 0, 0);
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

int pick_mb(int M, int K) {
  int mb = 1;
  while (mb < M && mb < 8) mb *= 2;
  return mb;
}

// K-chunk staged in LDS per pass: a multiple of the prefetch batch (512 * U elements)
int gv_kc(int mb) {
  const int step = 512 * (mb >= 8 ? 2 : 4);
  int kc = GV_LDS_FLOATS / mb;
  kc = (kc / step) * step;
  return kc < step ? step : kc;
}

template <typename WT>
hipError_t launch_gemv_t(const LinearArgs& a, hipStream_t s) {
  const bool gated = (a.epi == EPI_GATED_GELU || a.epi == EPI_GATED_SILU);
  const int n_total = gated ? a.n_per : a.n_per * a.n_mats;
  const int waves = gated ? a.n_per : (n_total + 1) / 2;
  const int mb = pick_mb(a.M, a.K);
  int kc = gv_kc(mb);
  if (a.K <= kc) kc = (a.K + 3) & ~3;  // one chunk: size the LDS to the row
  dim3 grid((waves + GV_WAVES - 1) / GV_WAVES, (a.M + mb - 1) / mb);
  const size_t shm = (size_t)mb * kc * sizeof(float);
  switch (mb) {
    case 1: hipLaunchKernelGGL((gemv_kernel<WT, 1>), grid, dim3(256), shm, s, a, kc); break;
    case 2: hipLaunchKernelGGL((gemv_kernel<WT, 2>), grid, dim3(256), shm, s, a, kc); break;
    case 4: hipLaunchKernelGGL((gemv_kernel<WT, 4>), grid, dim3(256), shm, s, a, kc); break;
    default: hipLaunchKernelGGL((gemv_kernel<WT, 8>), grid, dim3(256), shm, s, a, kc); break;
  }
  return hipGetLastError();
}

bool want_mfma(const LinearArgs& a) {
  if (a.wdtype != 1) return false;
  if (a.K % TK) return false;
  if (a.n_mats > 1 && a.n_per % TN) return false;  // tiles must not straddle matrices
  if (a.use_mfma >= 0) return a.use_mfma == 1;
  return a.M > 8;
}

}  // namespace

int argmax_parts(int n_out, int M, int wdtype) {
  LinearArgs a;
  a.M = M;
  a.wdtype = wdtype;
  if (want_mfma(a)) return (n_out + TN - 1) / TN;
  const int waves = (n_out + 1) / 2;
  return (waves + GV_WAVES - 1) / GV_WAVES;
}

hipError_t launch_row_stats(const float* x, int ldx, int M, int K, int norm, float eps,
                            float2* stats, hipStream_t s) {
  hipLaunchKernelGGL(row_stats_kernel, dim3(M), dim3(64), 0, s, x, ldx, M, K, norm, eps, stats);
  return hipGetLastError();
}

hipError_t launch_linear(LinearArgs a, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  const bool gated = (a.epi == EPI_GATED_GELU || a.epi == EPI_GATED_SILU);
  const int n_out = gated ? a.n_per : a.n_per * a.n_mats;
  if (want_mfma(a)) {
    a.use_mfma = 1;
    if (a.epi == EPI_ARGMAX) a.n_parts = (n_out + TN - 1) / TN;
    if (a.norm != NORM_NONE) {
      hipError_t e = launch_row_stats(a.x, a.ldx, a.M, a.K, a.norm, a.eps, a.stats, s);
      if (e != hipSuccess) return e;
    }
    dim3 grid((n_out + TN - 1) / TN, (a.M + TM - 1) / TM);
    if (gated) hipLaunchKernelGGL((gemm_kernel<true>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((gemm_kernel<false>), grid, dim3(256), 0, s, a);
    return hipGetLastError();
  }
  a.use_mfma = 0;
  if (a.epi == EPI_ARGMAX) a.n_parts = argmax_parts(n_out, a.M, 0);
  return a.wdtype == 1 ? launch_gemv_t<bf16_t>(a, s) : launch_gemv_t<float>(a, s);
}

}  // namespace ssd
