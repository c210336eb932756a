// Speculative sampling on the self-speculative loop: sampled draft tokens and the
// acceptance rule that keeps the full model's output distribution.
//
// Distributions at temperature tau: softmax(logits / tau).  Randomness is an input: a sample from
// weights w with uniform u is the inverse CDF, the smallest k with w_0 + ... + w_k > u * sum(w).
// A draft token x_i is accepted when u * q_i(x_i) < p_{i-1}(x_i) (probability min(1, p/q)); the
// first rejected position takes a sample from the normalised residual max(0, p - q) (p itself if
// it vanishes), and a round whose drafts all pass takes one more sample from p_gamma.
//
// One block of 256 threads per row (draft samples) or per sequence (acceptance).  Vocabulary
// sweeps are two passes (max, then the sum of exp((l - max) / tau)); the inverse CDF gives each
// thread a contiguous chunk of the vocabulary, scans the chunk sums across the block and walks
// the one chunk that holds the target.  Bound: a few passes over rows of V floats (L2-resident,
// just written by the LM head) and block synchronisation.
#include "device.h"
#include "kernels.h"

#include <climits>

namespace ssd {

namespace {

constexpr int SB = 256;  // threads per sampling block

__device__ float block_max(float v, float* red) {
  v = wave_max(v);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  const float r = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  __syncthreads();
  return r;
}

__device__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  const float r = (red[0] + red[1]) + (red[2] + red[3]);
  __syncthreads();
  return r;
}

// (max, sum of exp((l - max) / tau)) of a row of V logits
__device__ float2 row_norm(const float* row, int V, float inv_tau, float* red) {
  float m = -INFINITY;
  for (int j = threadIdx.x; j < V; j += SB) m = fmaxf(m, row[j]);
  m = block_max(m, red);
  float s = 0.f;
  for (int j = threadIdx.x; j < V; j += SB) s += __expf((row[j] - m) * inv_tau);
  s = block_sum(s, red);
  return make_float2(m, s);
}

// Inverse CDF over V weights weight(j) with uniform u: the smallest k with
// weight(0) + ... + weight(k) > u * total; past the total by rounding, the last index of positive
// weight.  Every thread of the block calls this; scan[] holds SB floats.
template <typename W>
__device__ int inverse_cdf(W weight, int V, float u, float* scan, int* pick) {
  const int tid = threadIdx.x, C = (V + SB - 1) / SB;
  const int j0 = min(V, tid * C), j1 = min(V, j0 + C);
  float s = 0.f;
  int last_pos = -1;
  for (int j = j0; j < j1; ++j) {
    const float w = weight(j);
    s += w;
    if (w > 0.f) last_pos = j;
  }
  scan[tid] = s;
  if (tid == 0) pick[0] = -1;
  __syncthreads();
  // inclusive scan of the chunk sums (Hillis-Steele)
  for (int off = 1; off < SB; off <<= 1) {
    const float v = tid >= off ? scan[tid - off] : 0.f;
    __syncthreads();
    scan[tid] += v;
    __syncthreads();
  }
  const float total = scan[SB - 1];
  const float target = u * total;
  const float before = tid ? scan[tid - 1] : 0.f;
  if (before <= target && target < scan[tid]) {
    float acc = before;
    int k = last_pos;
    for (int j = j0; j < j1; ++j) {
      acc += weight(j);
      if (acc > target) {
        k = j;
        break;
      }
    }
    pick[0] = k;
  }
  __syncthreads();
  int k = pick[0];
  __syncthreads();
  if (k < 0) {
    // target at or past the total (rounding): the last index of positive weight
    int lp = last_pos;
    for (int o = 32; o > 0; o >>= 1) lp = max(lp, __shfl_xor(lp, o, 64));
    if ((tid & 63) == 0) scan[tid >> 6] = __int_as_float(lp);
    __syncthreads();
    k = max(max(__float_as_int(scan[0]), __float_as_int(scan[1])),
            max(__float_as_int(scan[2]), __float_as_int(scan[3])));
    __syncthreads();
    if (k < 0) k = 0;
  }
  return k;
}

// Row m = b * C + j: sample from softmax(row / tau) with u[b * ldu + uoff + j]; token to
// dst0[b * ld0 + off0 + j] and dst1[m] (if set).
__global__ __launch_bounds__(SB) void sample_rows_kernel(const float* logits, int ldl, int V,
                                                         float inv_tau, const float* u, int ldu,
                                                         int uoff, int C, int32_t* dst0, int ld0,
                                                         int off0, int32_t* dst1) {
  __shared__ float red[4];
  __shared__ float scan[SB];
  __shared__ int pick[1];
  const int m = blockIdx.x, b = m / C, j = m - b * C;
  const float* row = logits + (size_t)m * ldl;
  const float2 n = row_norm(row, V, inv_tau, red);
  const float uu = u[(size_t)b * ldu + uoff + j];
  const int k = inverse_cdf([&](int i) { return __expf((row[i] - n.x) * inv_tau); }, V, uu, scan,
                            pick);
  if (threadIdx.x == 0) {
    dst0[(size_t)b * ld0 + off0 + j] = k;
    if (dst1) dst1[m] = k;
  }
}

__global__ __launch_bounds__(SB) void accept_sample_kernel(const AcceptSampleArgs a) {
  __shared__ float red[4];
  __shared__ float scan[SB];
  __shared__ int pick[1];
  const int b = blockIdx.x, g = a.gamma, V = a.vocab;
  if (a.active && a.active[b] == 0) return;
  const float it = a.inv_tau;
  const int32_t* dr = a.draft + (size_t)b * g;
  const float* ub = a.u + (size_t)b * (g + 1);
  int acc = g, tok = 0;
  for (int i = 0; i < g; ++i) {
    const float* P = a.target_logits + ((size_t)b * (g + 1) + i) * V;
    const float* Q = a.draft_logits + ((size_t)b * g + i) * V;
    const float2 np_ = row_norm(P, V, it, red);
    const float2 nq = row_norm(Q, V, it, red);
    int x = dr[i];
    if (x < 0 || x >= V) x = 0;  // out-of-range drafts never pass (q(x) is set below)
    const float px = __expf((P[x] - np_.x) * it) / np_.y;
    const float qx = dr[i] == x ? __expf((Q[x] - nq.x) * it) / nq.y : INFINITY;
    if (ub[i] * qx < px) continue;
    acc = i;
    const float ip = 1.0f / np_.y, iq = 1.0f / nq.y;
    auto resid = [&](int j) {
      return fmaxf(__expf((P[j] - np_.x) * it) * ip - __expf((Q[j] - nq.x) * it) * iq, 0.f);
    };
    // the residual vanishes only when p = q: then p itself
    float rs = 0.f;
    for (int j = threadIdx.x; j < V; j += SB) rs += resid(j);
    rs = block_sum(rs, red);
    if (rs > 0.f)
      tok = inverse_cdf(resid, V, ub[g], scan, pick);
    else
      tok = inverse_cdf([&](int j) { return __expf((P[j] - np_.x) * it); }, V, ub[g], scan, pick);
    break;
  }
  if (acc == g) {
    const float* P = a.target_logits + ((size_t)b * (g + 1) + g) * V;
    const float2 np_ = row_norm(P, V, it, red);
    tok = inverse_cdf([&](int j) { return __expf((P[j] - np_.x) * it); }, V, ub[g], scan, pick);
  }
  if (threadIdx.x == 0) {
    if (a.out) {
      int32_t* o = a.out + (size_t)b * (g + 1);
      for (int i = 0; i < acc; ++i) o[i] = dr[i];
      o[acc] = tok;
    }
    if (a.accept_len) a.accept_len[b] = acc;
    a.pending[b] = tok;
    const int sl = a.seq_len[b] + acc + 1;
    a.seq_len[b] = sl;
    if (sl > a.max_seq) atomicOr(a.status, SSD_DEV_CAPACITY);
  }
}

}  // namespace

hipError_t launch_sample_rows(const float* logits, int ldl, int M, int V, float tau,
                              const float* u, int ldu, int uoff, int C, int32_t* dst0, int ld0,
                              int off0, int32_t* dst1, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  hipLaunchKernelGGL(sample_rows_kernel, dim3(M), dim3(SB), 0, s, logits, ldl, V, 1.0f / tau, u,
                     ldu, uoff, C, dst0, ld0, off0, dst1);
  return hipGetLastError();
}

hipError_t launch_accept_sample(const AcceptSampleArgs& a, hipStream_t s) {
  if (a.B <= 0) return hipSuccess;
  hipLaunchKernelGGL(accept_sample_kernel, dim3(a.B), dim3(SB), 0, s, a);
  return hipGetLastError();
}

}  // namespace ssd
