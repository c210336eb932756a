// Small kernels of the decode loop: input gather, rotary + KV scatter, argmax reduction, greedy
// acceptance with KV-length rollback, and generation bookkeeping.
#include "device.h"
#include "kernels.h"

#include <climits>

namespace ssd {

namespace {

template <typename WT>
__global__ void embed_kernel(const EmbedArgs a) {
  const int r = blockIdx.x;
  const int b = r / a.C, j = r - b * a.C;
  float* xr = a.x + (size_t)r * a.d;
  const WT* src;
  if (j < a.n_prefix) {
    src = reinterpret_cast<const WT*>(a.visual) + ((size_t)b * a.n_visual + j) * a.d;
  } else {
    const int jj = j - a.n_prefix;
    int tok = (a.t0 && jj == 0) ? a.t0[b] : a.t1[(size_t)b * a.ld1 + jj - (a.t0 ? 1 : 0)];
    if (tok < 0 || tok >= a.vocab) {
      if (threadIdx.x == 0) atomicOr(a.status, SSD_DEV_BAD_TOKEN);
      tok = 0;
    }
    src = reinterpret_cast<const WT*>(a.embed) + (size_t)tok * a.d;
  }
  for (int k = threadIdx.x; k < a.d; k += blockDim.x) xr[k] = load_elem(src + k);
}

template <typename KT>
__global__ void rope_scatter_kernel(const RopeScatterArgs a) {
  const int r = blockIdx.x;
  const int b = r / a.C, j = r - b * a.C;
  const int HD = a.H * a.dh, half = a.dh / 2;
  const int pos = a.kv.seq_len[b] + a.kv.pos_off + j;
  int page = -1;
  const int pg_i = pos >= 0 ? pos / a.kv.page_size : -1;
  if (pos < 0 || pos >= a.max_seq || pg_i >= a.kv.max_pages) {
    if (threadIdx.x == 0) atomicOr(a.status, SSD_DEV_CAPACITY);
  } else {
    page = a.kv.page_table[(size_t)b * a.kv.max_pages + pg_i];
    if (page < 0 || page >= a.kv.n_pages) {
      if (threadIdx.x == 0) atomicOr(a.status, SSD_DEV_BAD_PAGE);
      page = -1;
    }
  }
  const int slot = pos - pg_i * a.kv.page_size;
  const int tpos = pos < 0 ? 0 : (pos >= a.max_seq ? a.max_seq - 1 : pos);
  const float* src = a.qkv + (size_t)r * 3 * HD;
  for (int idx = threadIdx.x; idx < a.H * half; idx += blockDim.x) {
    const int h = idx / half, i = idx - h * half;
    const int c0 = h * a.dh + i, c1 = c0 + half;
    float q0 = src[c0], q1 = src[c1];
    float k0 = src[HD + c0], k1 = src[HD + c1];
    const float v0 = src[2 * HD + c0], v1 = src[2 * HD + c1];
    if (a.rope_cos) {
      const float cs = a.rope_cos[(size_t)tpos * half + i], sn = a.rope_sin[(size_t)tpos * half + i];
      const float rq0 = q0 * cs - q1 * sn, rq1 = q1 * cs + q0 * sn;
      const float rk0 = k0 * cs - k1 * sn, rk1 = k1 * cs + k0 * sn;
      q0 = rq0; q1 = rq1; k0 = rk0; k1 = rk1;
    }
    a.q_out[(size_t)r * HD + c0] = q0;
    a.q_out[(size_t)r * HD + c1] = q1;
    if (page >= 0) {
      const size_t off = (((size_t)page * a.H + h) * a.kv.page_size + slot) * a.dh;
      KT* kp = reinterpret_cast<KT*>(a.kv.k) + off;
      KT* vp = reinterpret_cast<KT*>(a.kv.v) + off;
      store_elem(kp + i, k0);
      store_elem(kp + i + half, k1);
      store_elem(vp + i, v0);
      store_elem(vp + i + half, v1);
    }
  }
}

template <typename WT>
__global__ __launch_bounds__(256) void argmax_final_kernel(const float* pv, const int* pi, int M,
                                                           int n_parts, int C, int32_t* dst0,
                                                           int ld0, int off0, int32_t* dst1,
                                                           const WT* embed, int d, float* x_out,
                                                           const ConfArgs cf) {
  constexpr int PER = 16;  // partials per thread requested together
  __shared__ float sv[4];
  __shared__ int si[4];
  __shared__ int tok;
  __shared__ float vmax;
  const int m = blockIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  float v = -INFINITY;
  int i = INT_MAX;
  for (int p0 = 0; p0 < n_parts; p0 += 256 * PER) {
    float vv[PER];
    int ii[PER];
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int p = p0 + u * 256 + threadIdx.x;
      vv[u] = p < n_parts ? pv[(size_t)m * n_parts + p] : -INFINITY;
      ii[u] = p < n_parts ? pi[(size_t)m * n_parts + p] : INT_MAX;
    }
#pragma unroll
    for (int u = 0; u < PER; ++u) argmax_merge(v, i, vv[u], ii[u]);
  }
  wave_argmax(v, i);
  if (lane == 0) { sv[wave] = v; si[wave] = i; }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < (int)(blockDim.x >> 6); ++w) argmax_merge(v, i, sv[w], si[w]);
    if (i == INT_MAX) i = 0;  // every logit NaN: nothing sensible to choose
    const int b = m / C, j = m - b * C;
    dst0[(size_t)b * ld0 + off0 + j] = i;
    if (dst1) dst1[m] = i;
    tok = i;
    vmax = v;
  }
  if (cf.logits) {
    // confidence: 1 / sum_n exp(logit_n - max) over the row
    __syncthreads();
    const float mx = vmax;
    const float* row = cf.logits + (size_t)m * cf.ldl;
    float s = 0.f;
    for (int n = threadIdx.x; n < cf.V; n += blockDim.x) s += expf(row[n] - mx);
    s = wave_sum(s);
    __syncthreads();
    if (lane == 0) sv[wave] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
      float tot = 0.f;
      for (int w = 0; w < (int)(blockDim.x >> 6); ++w) tot += sv[w];
      const float conf = 1.0f / tot;
      if (cf.conf) cf.conf[(size_t)m * cf.ldc + cf.step] = conf;
      const bool act = !cf.active || cf.active[m] != 0;
      if (cf.step == 0) {
        cf.ndraft[m] = act ? 1 : 0;
        cf.drafting[m] = (act && conf >= cf.tau) ? 1 : 0;
      } else if (cf.drafting[m]) {
        cf.ndraft[m] = cf.step + 1;
        cf.drafting[m] = conf >= cf.tau ? 1 : 0;
      }
    }
  }
  if (!x_out) return;
  // the chosen token's embedding row, the next draft step's input (row m of x_out)
  __syncthreads();
  const WT* src = embed + (size_t)tok * d;
  for (int k = threadIdx.x; k < d; k += blockDim.x) x_out[(size_t)m * d + k] = load_elem(src + k);
}

// Read-only stream: block b reads the 16 KB chunk b of n16 16-byte words, four loads in flight
// per thread (the form that streamed fastest among grid-stride and 16-128 KB chunk variants on
// MI355X).  out[b % 4096] is written only when the XOR of the chunk hits a fixed word, which the
// compiler cannot rule out, so the loads are kept.
__global__ __launch_bounds__(256) void read_probe_kernel(const uint4* __restrict__ p, size_t n16,
                                                         float* out) {
  constexpr size_t CHUNK = 1024;  // 16-byte words per block
  const size_t base = (size_t)blockIdx.x * CHUNK;
  uint32_t acc = 0;
  uint4 v[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const size_t j = base + (size_t)u * 256 + threadIdx.x;
    v[u] = j < n16 ? p[j] : make_uint4(0, 0, 0, 0);
  }
#pragma unroll
  for (int u = 0; u < 4; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  if (acc == 0x9e3779b9u) out[blockIdx.x & 4095] = 1.f;
}

__global__ void copy_tokens_kernel(int32_t* dst, int ld_dst, const int32_t* src, int ld_src,
                                   int B, int n) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= B * n) return;
  const int b = e / n, j = e - b * n;
  dst[(size_t)b * ld_dst + j] = src[(size_t)b * ld_src + j];
}

template <typename KT>
__global__ void scatter_cross_kernel(const float* src, KT* dst, int B, int Nv, int H, int dh) {
  const int r = blockIdx.x;  // b * Nv + n
  const int b = r / Nv, n = r - b * Nv;
  const int HD = H * dh;
  for (int c = threadIdx.x; c < HD; c += blockDim.x) {
    const int h = c / dh, d = c - h * dh;
    store_elem(dst + (((size_t)b * H + h) * Nv + n) * dh + d, src[(size_t)r * HD + c]);
  }
}

__global__ void assemble_kernel(float* x, const float* stash, int ld_stash_b, const float* x1,
                                int B, int g, int d) {
  const int r = blockIdx.x;  // b * (g + 1) + j
  const int b = r / (g + 1), j = r - b * (g + 1);
  const float* src = j < g ? stash + (size_t)b * ld_stash_b + (size_t)j * d : x1 + (size_t)b * d;
  for (int k = threadIdx.x; k < d; k += blockDim.x) x[(size_t)r * d + k] = src[k];
}

// dst row r (stride ldd) = src row r (stride lds), cols floats each; one block per row
__global__ void copy_rows_kernel(float* dst, int ldd, const float* src, int lds, int cols) {
  const size_t r = blockIdx.x;
  for (int k = threadIdx.x; k < cols; k += blockDim.x) dst[r * ldd + k] = src[r * lds + k];
}

__global__ void set_seq_len_kernel(int32_t* seq_len, int B, int value) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b < B) seq_len[b] = value;
}

__global__ void accept_kernel(const AcceptArgs a) {
  __shared__ int acc_n[256];
  __shared__ int act_after[256];
  __shared__ int len_after[256];
  __shared__ int need_after[256];
  __shared__ int prop_n[256];
  const int b = threadIdx.x;
  const int g = a.gamma;
  int n = 0;
  int still = 0;
  bool did = false;
  if (b < a.B) {
    bool act = a.active ? (a.active[b] != 0) : true;
    if (a.active_rw) act = act && (a.active_rw[b] != 0);
    if (act) {
      did = true;
      const int32_t* dr = a.draft + (size_t)b * g;
      const int32_t* tg = a.target + (size_t)b * (g + 1);
      // drafts this sequence proposed this round (confidence-stopped drafting: fewer than g)
      const int gb = a.ndraft ? max(0, min(g, a.ndraft[b])) : g;
      while (n < gb && dr[n] == tg[n]) ++n;
      if (a.out) {
        int32_t* o = a.out + (size_t)b * (g + 1);
        for (int i = 0; i < n; ++i) o[i] = dr[i];
        o[n] = tg[n];
      }
      if (a.accept_len) a.accept_len[b] = n;
      int adv = n + 1;
      a.pending[b] = tg[n];
      still = 1;
      if (a.tokens) {
        const int c = a.count[b];
        const int emit = min(n + 1, a.T - c);
        for (int e = 0; e < emit; ++e) a.tokens[(size_t)b * a.T + c + e] = e < n ? dr[e] : tg[n];
        a.count[b] = c + emit;
        if (c + emit >= a.T) {
          // finished: keep only the emitted positions, so the rows this sequence still occupies
          // in later rounds of the batch stay inside the cache
          adv = emit;
          a.active_rw[b] = 0;
          still = 0;
        }
      }
      const int sl = a.seq_len[b] + adv;
      a.seq_len[b] = sl;
      if (sl + (still ? a.next_need : 0) > a.max_seq) atomicOr(a.status, SSD_DEV_CAPACITY);
    } else if (a.active_rw) {
      still = 0;
    }
  }
  acc_n[b] = did ? n : -1;
  prop_n[b] = did ? (a.ndraft ? max(0, min(g, a.ndraft[b])) : g) : 0;
  act_after[b] = still;
  len_after[b] = (b < a.B && still) ? a.seq_len[b] : INT_MAX;
  need_after[b] = (b < a.B && still && a.tokens) ? a.T - a.count[b] : 0;
  __syncthreads();
  if (b == 0 && a.stats) {
    long long sa = 0, sd = 0;
    int na = 0, lmin = INT_MAX, need = 0;
    for (int t = 0; t < a.B && t < 256; ++t) {
      if (acc_n[t] >= 0) { sa += acc_n[t]; sd += prop_n[t]; }
      na += act_after[t];
      lmin = min(lmin, len_after[t]);
      need = max(need, need_after[t]);
    }
    a.stats[0] += 1;
    a.stats[1] += sa;
    a.stats[2] += sd;
    if (a.n_active) {
      a.n_active[0] = na;
      a.n_active[1] = na ? lmin : 0;
      a.n_active[3] = need;
      // the device status word (an atomic read: the bits come from atomics of this and
      // earlier launches)
      a.n_active[2] = a.status ? atomicOr(a.status, 0) : 0;
    }
  }
}

__global__ void gen_init_kernel(const GenInitArgs a) {
  __shared__ int act[256];
  const int b = threadIdx.x;
  act[b] = 0;
  if (b < a.B) {
    a.tokens[(size_t)b * a.T] = a.pending[b];
    a.count[b] = 1;
    a.active[b] = a.T > 1 ? 1 : 0;
    act[b] = a.active[b];
  }
  __syncthreads();
  if (b == 0) {
    int na = 0, lmin = INT_MAX;
    for (int t = 0; t < a.B && t < 256; ++t) {
      na += act[t];
      if (act[t]) lmin = min(lmin, a.seq_len[t]);
    }
    a.n_active[0] = na;
    a.n_active[1] = na ? lmin : 0;
    a.n_active[2] = a.status ? atomicOr(a.status, 0) : 0;
    a.n_active[3] = na ? a.T - 1 : 0;  // tokens the longest-running sequence still needs
    a.stats[0] = a.stats[1] = a.stats[2] = 0;
  }
}

__global__ void bias_table_kernel(const float* rel_bias, const int32_t* bucket, int H, int max_seq,
                                  float* table) {
  const int n = blockIdx.x * blockDim.x + threadIdx.x;
  if (n >= max_seq) return;
  const int bk = bucket[n];
  for (int h = 0; h < H; ++h) table[(size_t)h * max_seq + n] = rel_bias[(size_t)bk * H + h];
}

}  // namespace

hipError_t launch_embed(const EmbedArgs& a, hipStream_t s) {
  if (a.B * a.C <= 0) return hipSuccess;
  if (a.wdtype == 1) hipLaunchKernelGGL(embed_kernel<bf16_t>, dim3(a.B * a.C), dim3(256), 0, s, a);
  else hipLaunchKernelGGL(embed_kernel<float>, dim3(a.B * a.C), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_rope_scatter(const RopeScatterArgs& a, hipStream_t s) {
  if (a.B * a.C <= 0) return hipSuccess;
  if (a.kvdtype == 1) hipLaunchKernelGGL(rope_scatter_kernel<bf16_t>, dim3(a.B * a.C), dim3(256), 0, s, a);
  else hipLaunchKernelGGL(rope_scatter_kernel<float>, dim3(a.B * a.C), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_argmax_final_ex(const float* part_val, const int* part_idx, int M, int n_parts,
                                  int C, int32_t* dst0, int ld0, int off0, int32_t* dst1,
                                  const void* embed, int wdtype, int d, float* x_out,
                                  const ConfArgs& cf, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  if (x_out && (!embed || d < 1)) return hipErrorInvalidValue;
  if (cf.logits && (!cf.drafting || !cf.ndraft || cf.V < 1)) return hipErrorInvalidValue;
  if (x_out && wdtype == 1)
    hipLaunchKernelGGL(argmax_final_kernel<bf16_t>, dim3(M), dim3(256), 0, s, part_val, part_idx,
                       M, n_parts, C, dst0, ld0, off0, dst1,
                       reinterpret_cast<const bf16_t*>(embed), d, x_out, cf);
  else
    hipLaunchKernelGGL(argmax_final_kernel<float>, dim3(M), dim3(256), 0, s, part_val, part_idx,
                       M, n_parts, C, dst0, ld0, off0, dst1,
                       x_out ? reinterpret_cast<const float*>(embed) : nullptr, d, x_out, cf);
  return hipGetLastError();
}

hipError_t launch_argmax_final(const float* part_val, const int* part_idx, int M, int n_parts,
                               int C, int32_t* dst0, int ld0, int off0, int32_t* dst1,
                               hipStream_t s) {
  return launch_argmax_final_ex(part_val, part_idx, M, n_parts, C, dst0, ld0, off0, dst1,
                                nullptr, 0, 0, nullptr, ConfArgs(), s);
}

hipError_t launch_argmax_final_embed(const float* part_val, const int* part_idx, int M,
                                     int n_parts, int C, int32_t* dst0, int ld0, int off0,
                                     int32_t* dst1, const void* embed, int wdtype, int d,
                                     float* x_out, hipStream_t s) {
  if (!embed || !x_out || d < 1) return hipErrorInvalidValue;
  return launch_argmax_final_ex(part_val, part_idx, M, n_parts, C, dst0, ld0, off0, dst1, embed,
                                wdtype, d, x_out, ConfArgs(), s);
}

hipError_t launch_read_probe(const void* buf, size_t bytes, float* out, hipStream_t s) {
  if (bytes < 16) return hipErrorInvalidValue;
  const size_t blocks = (bytes / 16 + 1023) / 1024;
  if (blocks > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL(read_probe_kernel, dim3((unsigned)blocks), dim3(256), 0, s,
                     reinterpret_cast<const uint4*>(buf), bytes / 16, out);
  return hipGetLastError();
}

hipError_t launch_copy_tokens(int32_t* dst, int ld_dst, const int32_t* src, int ld_src, int B,
                              int n, hipStream_t s) {
  if (B * n <= 0) return hipSuccess;
  hipLaunchKernelGGL(copy_tokens_kernel, dim3((B * n + 255) / 256), dim3(256), 0, s, dst, ld_dst,
                     src, ld_src, B, n);
  return hipGetLastError();
}

hipError_t launch_scatter_cross(const float* src, void* dst, int B, int Nv, int H, int dh,
                                int kvdtype, hipStream_t s) {
  if (B * Nv <= 0) return hipSuccess;
  if (kvdtype == 1)
    hipLaunchKernelGGL(scatter_cross_kernel<bf16_t>, dim3(B * Nv), dim3(256), 0, s, src,
                       reinterpret_cast<bf16_t*>(dst), B, Nv, H, dh);
  else
    hipLaunchKernelGGL(scatter_cross_kernel<float>, dim3(B * Nv), dim3(256), 0, s, src,
                       reinterpret_cast<float*>(dst), B, Nv, H, dh);
  return hipGetLastError();
}

hipError_t launch_assemble(float* x, const float* stash, int ld_stash_b, const float* x1, int B,
                           int g, int d, hipStream_t s) {
  hipLaunchKernelGGL(assemble_kernel, dim3(B * (g + 1)), dim3(256), 0, s, x, stash, ld_stash_b, x1,
                     B, g, d);
  return hipGetLastError();
}

hipError_t launch_copy_rows(float* dst, int ldd, const float* src, int lds, int rows, int cols,
                            hipStream_t s) {
  if (rows <= 0 || cols <= 0) return hipSuccess;
  hipLaunchKernelGGL(copy_rows_kernel, dim3(rows), dim3(256), 0, s, dst, ldd, src, lds, cols);
  return hipGetLastError();
}

hipError_t launch_set_seq_len(int32_t* seq_len, int B, int value, hipStream_t s) {
  hipLaunchKernelGGL(set_seq_len_kernel, dim3((B + 255) / 256), dim3(256), 0, s, seq_len, B, value);
  return hipGetLastError();
}

hipError_t launch_accept(const AcceptArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(accept_kernel, dim3(1), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_gen_init(const GenInitArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(gen_init_kernel, dim3(1), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_bias_table(const float* rel_bias, const int32_t* bucket, int H, int max_seq,
                             float* table, hipStream_t s) {
  hipLaunchKernelGGL(bias_table_kernel, dim3((max_seq + 255) / 256), dim3(256), 0, s, rel_bias,
                     bucket, H, max_seq, table);
  return hipGetLastError();
}

}  // namespace ssd
