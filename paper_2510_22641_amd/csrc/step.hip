// Persistent one-row pass of the decoder for one sequence: a whole draft step (layers 1..k, the
// imitation network, g and the argmax), a greedy step (all layers, g, argmax) or the one-row part
// of a verify that reuses the draft's layer-k states, as ONE launch of one block per compute unit.
//
// A batch-1 step is a chain of dependent matrix-vector products: every product's output feeds a
// norm over the whole row, so a chain of separate kernels pays one launch (a few microseconds of
// ramp-up, drain and dispatch) per product, which at the FlanT5-xl shape costs more than the
// weight bytes themselves.  Here the pass is a list of phases built on the host (StepPhase):
//   SP_GEMV     y = epilogue(W . transform(x)): weight rows streamed in pairs by 7 compute waves
//               per block, the input row staged once per block in LDS by the eighth wave;
//   SP_ATTN     self-attention of the row's query over the paged cache, split over keys
//               (one wave per (head, key split), writing (output, max, sum) partials);
//   SP_COMBINE  merge of many key-split partials into the attention output.
// Phases are separated by a grid barrier.  After its outputs of a phase are complete, a block
// publishes a flag; one wave per block polls every block's flag.  Before waiting, each compute
// wave requests the weights of its first row pair of the next phase (weights never depend on the
// activations), so the weight stream continues through the barrier.
//
// Visibility across the XCDs (each has its own L2): everything another block reads within the
// launch is written with agent-scope (sc1) stores, and a block publishes its flag only after its
// stores have completed; flags are read with sc1 loads.  Each phase writes to addresses that no
// block reads before that phase's barrier, and no activation or cache entry is written twice
// within a launch, so no cache holds an outdated copy of a value when it is read (caches are
// invalidated between launches, as for any pair of kernels).
//
// Every wait is bounded: past the spin limit the block sets SSD_DEV_SYNC and an abort word that
// every waiter checks, and leaves; a launch that finds the abort word set leaves at once.
//
// Measured on MI355X this pass is slower than the chain of kernels it replaces (FlanT5-xl draft
// step 562 us against 367 us; LLaVA-7B 1582 us against 926 us), so it is off by default.  Under
// the weight stream a memory round trip takes 3-4 us, and each phase pays about three of them in
// series (the flags, the staged input row, the acknowledgement of its own stores): barrier plus
// staging cost about 5.5 us per phase against about 2 us for a kernel boundary, while the
// phases' streaming, with one chunk per wave in flight, is no faster than the one-shot kernels.
#include "device.h"
#include "kernels.h"

#include <hip/hip_ext.h>

#include <climits>

namespace ssd {

namespace {

constexpr int ST_WAVES = 8;
constexpr int ST_CW = 7;  // compute waves; wave 7 polls the flags and stages the inputs
constexpr int ST_THREADS = 64 * ST_WAVES;
constexpr int XS_HALF = STEP_XS_MAX / 2;
constexpr int REC = 4;  // a partial record is dh outputs, max, sum, 2 pad floats (16-byte rows)

typedef float f32x4_t_ __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t_ __attribute__((ext_vector_type(4)));

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc_of(const void* p) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), 0, 0x7fffffff, 0x00020000);
}

// agent-coherent stores and loads (sc1): seen by every XCD once complete
__device__ __forceinline__ void st_coh(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_coh(int* p, int v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_coh(uint32_t* p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_coh(bf16_t* p, float v) {
  __hip_atomic_store(p, (bf16_t)f32_to_bf16(v), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_coh4(float* p, float a, float b, float c, float d) {
  f32x4_t_ v = {a, b, c, d};
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4_t_, v), rsrc_of(p), 0, 0, 16);
}
__device__ __forceinline__ uint32_t ld_coh(const uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Split-plane LDS layout of a staged row: element k sits in plane (k / 4) % 2 at
// (k / 8) * 4 + k % 4, so the two 16-byte reads of a lane's 8 consecutive elements are each
// contiguous across the wave.
__device__ __forceinline__ void xs_put8(float* xs, int g, const float* v) {
  *reinterpret_cast<float4*>(xs + g * 4) = make_float4(v[0], v[1], v[2], v[3]);
  *reinterpret_cast<float4*>(xs + XS_HALF + g * 4) = make_float4(v[4], v[5], v[6], v[7]);
}
__device__ __forceinline__ void xs_get8(const float* xs, int g, float* v) {
  const float4 a = *reinterpret_cast<const float4*>(xs + g * 4);
  const float4 b = *reinterpret_cast<const float4*>(xs + XS_HALF + g * 4);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}

__device__ __forceinline__ void load8(const float* p, float* v) {
  const float4 a = reinterpret_cast<const float4*>(p)[0];
  const float4 b = reinterpret_cast<const float4*>(p)[1];
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}
__device__ __forceinline__ void load8(const bf16_t* p, float* v) {
  unpack_bf16x8(*reinterpret_cast<const uint4*>(p), v);
}

// ---------------------------------------------------------------------------------------------
// Grid barrier: wave 7 of every block waits until every block has published phase `want`.

__device__ bool poll_flags(const StepArgs& a, uint32_t want, int lane, int nblk) {
  uint32_t spins = 0;
  while (true) {
    bool mine = true;
    for (int b0 = 0; b0 < nblk; b0 += 256) {
      const int idx = b0 + lane * 4;
      if (idx < nblk) {
        const u32x4_t_ f = __builtin_bit_cast(
            u32x4_t_, __builtin_amdgcn_raw_buffer_load_b128(rsrc_of(a.flags), idx * 4, 0, 16));
#pragma unroll
        for (int j = 0; j < 4; ++j)
          if (idx + j < nblk) mine = mine && (int)(f[j] - want) >= 0;
      }
    }
    if (__all(mine)) return true;
    if (ld_coh(a.abort_word) != 0u) return false;
    if (++spins > a.spin_limit) {
      if (lane == 0) {
        st_coh(a.abort_word, 1u);
        atomicOr(a.status, SSD_DEV_SYNC);
      }
      return false;
    }
  }
}

// ---------------------------------------------------------------------------------------------
// Input staging (wave 7 alone for a plain or embedded row; the whole block for attention
// partials).  Leaves transform(x) in xs (zero past K up to a multiple of 2048), the raw row in
// xres when it is the residual, and in *nscale the factor that multiplies every dot product
// (1/rms for RMSNorm, whose gain is already applied in xs; 1 otherwise).

template <typename ET>
__device__ void stage_row(const StepPhase& ph, const ET* src, float* xs, float* xres,
                          float* nscale, int lane) {
  const int K = ph.K;
  const int nsl = (K + 2047) / 2048;
  const int norm = ph.norm;
  float s1 = 0.f, s2 = 0.f;
  for (int sl = 0; sl < nsl; ++sl) {
    float xv[4][8], gv[4][8];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int g = sl * 256 + i * 64 + lane;
      if (g * 8 < K) {
        load8(src + g * 8, xv[i]);
        if (norm == NORM_RMS || norm == NORM_LN) load8(ph.gain + g * 8, gv[i]);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) xv[i][e] = 0.f;
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int g = sl * 256 + i * 64 + lane;
      const bool live = g * 8 < K;
      if (ph.in_resid && live) {
        *reinterpret_cast<float4*>(xres + g * 8) = make_float4(xv[i][0], xv[i][1], xv[i][2], xv[i][3]);
        *reinterpret_cast<float4*>(xres + g * 8 + 4) = make_float4(xv[i][4], xv[i][5], xv[i][6], xv[i][7]);
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        s1 += xv[i][e];
        s2 = fmaf(xv[i][e], xv[i][e], s2);
      }
      float o[8];
      if (norm == NORM_RMS && live) {
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] = xv[i][e] * gv[i][e];
      } else if (norm == NORM_SOFTMAX) {
        // groups of ph.group consecutive inputs: group / 8 lanes each (aligned)
        float m = -INFINITY;
#pragma unroll
        for (int e = 0; e < 8; ++e) m = fmaxf(m, xv[i][e]);
        for (int off = 1; off < ph.group / 8; off <<= 1) m = fmaxf(m, __shfl_xor(m, off, 64));
        float sum = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          o[e] = live ? __expf(xv[i][e] - m) : 0.f;
          sum += o[e];
        }
        for (int off = 1; off < ph.group / 8; off <<= 1) sum += __shfl_xor(sum, off, 64);
        const float inv = live ? 1.0f / sum : 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] *= inv;
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] = xv[i][e];
      }
      xs_put8(xs, g, o);
    }
  }
  float scale = 1.f;
  if (norm == NORM_RMS) {
    s2 = wave_sum(s2);
    scale = 1.0f / sqrtf(s2 / (float)K + ph.eps);
  } else if (norm == NORM_LN) {
    const float mean = wave_sum(s1) / (float)K;
    float v2 = 0.f;
    for (int g = lane; g * 8 < K; g += 64) {
      float v[8];
      xs_get8(xs, g, v);
#pragma unroll
      for (int e = 0; e < 8; ++e) v2 = fmaf(v[e] - mean, v[e] - mean, v2);
    }
    const float rstd = 1.0f / sqrtf(wave_sum(v2) / (float)K + ph.eps);
    for (int g = lane; g * 8 < K; g += 64) {
      float v[8], gg[8], bb[8];
      xs_get8(xs, g, v);
      load8(ph.gain + g * 8, gg);
      load8(ph.shift + g * 8, bb);
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = (v[e] - mean) * rstd * gg[e] + bb[e];
      xs_put8(xs, g, v);
    }
  }
  if (lane == 0) *nscale = scale;
}

// Attention partials [H][S][dh + 4] -> the merged attention output in xs (whole block, S small).
__device__ void stage_attn(const StepPhase& ph, float* xs, int tid, int dh) {
  const int S = ph.n_splits, K = ph.K;
  for (int g = tid; g * 8 < K; g += ST_THREADS) {
    const int k = g * 8, h = k / dh, e0 = k - h * dh;
    const float* rec = ph.x + (size_t)h * S * (dh + REC);
    float mx[STEP_INLINE_SPLITS], ls[STEP_INLINE_SPLITS], ov[STEP_INLINE_SPLITS][8];
#pragma unroll
    for (int s = 0; s < STEP_INLINE_SPLITS; ++s) {
      if (s < S) {
        const float* r = rec + (size_t)s * (dh + REC);
        mx[s] = r[dh];
        ls[s] = r[dh + 1];
        load8(r + e0, ov[s]);
      }
    }
    float M = -INFINITY;
#pragma unroll
    for (int s = 0; s < STEP_INLINE_SPLITS; ++s)
      if (s < S) M = fmaxf(M, mx[s]);
    float L = 0.f, o[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < STEP_INLINE_SPLITS; ++s) {
      if (s < S) {
        const float wgt = mx[s] == -INFINITY ? 0.f : __expf(mx[s] - M);
        L = fmaf(wgt, ls[s], L);
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] = fmaf(wgt, ov[s][e], o[e]);
      }
    }
    const float inv = 1.0f / L;
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] *= inv;
    xs_put8(xs, g, o);
  }
  // zero tail up to a multiple of 2048
  const int Kpad = (K + 2047) / 2048 * 2048;
  for (int g = K / 8 + tid; g * 8 < Kpad; g += ST_THREADS) {
    float z[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    xs_put8(xs, g, z);
  }
}

// ---------------------------------------------------------------------------------------------
// GEMV tasks: a task is a row pair (two consecutive rows, the rotary pair (i, i + dh/2) of one
// head for QKV, or the (gate, up) rows of one feature); its K range is read in chunks of 4 KB per
// row (2048 bf16 or 1024 float32 elements), 64 bytes per lane per row.

struct Chunk {
  uint4 r0[4], r1[4];
};

struct TaskRows {
  const void* w0;
  const void* w1;
  int n0, n1;
  bool ok1;
  int mat;  // QKV: 0 q, 1 k, 2 v
  int c0;   // QKV: column of the pair's first element within its matrix
};

__device__ __forceinline__ TaskRows task_rows(const StepPhase& ph, int t, int esz, int d_head) {
  TaskRows r;
  const size_t rowb = (size_t)ph.K * esz;
  r.mat = 0;
  r.c0 = 0;
  if (ph.epi == EPI_GATED_GELU || ph.epi == EPI_GATED_SILU) {
    r.n0 = r.n1 = t;
    r.ok1 = true;
    r.w0 = (const char*)ph.w[0] + (size_t)t * rowb;
    r.w1 = (const char*)ph.w[1] + (size_t)t * rowb;
    return r;
  }
  if (ph.epi == EPI_QKV) {
    const int hd2 = ph.n_per >> 1, half = d_head >> 1;
    const int mat = t >= hd2 ? (t >= 2 * hd2 ? 2 : 1) : 0;
    const int loc = t - mat * hd2;
    const int h = loc / half, i = loc - h * half;
    const int c0 = h * d_head + i;
    r.mat = mat;
    r.c0 = c0;
    r.n0 = mat * ph.n_per + c0;
    r.n1 = r.n0 + half;
    r.ok1 = true;
    const void* base = mat == 0 ? ph.w[0] : (mat == 1 ? ph.w[1] : ph.w[2]);
    r.w0 = (const char*)base + (size_t)c0 * rowb;
    r.w1 = (const char*)r.w0 + (size_t)half * rowb;
    return r;
  }
  const int n_total = ph.n_per * ph.n_mats;
  r.n0 = 2 * t;
  r.n1 = 2 * t + 1;
  r.ok1 = r.n1 < n_total;
  int v0 = r.n0, v1 = r.ok1 ? r.n1 : r.n0;
  const void* b0 = ph.w[0];
  if (v0 >= ph.n_per) { v0 -= ph.n_per; b0 = ph.w[1]; if (v0 >= ph.n_per) { v0 -= ph.n_per; b0 = ph.w[2]; } }
  const void* b1 = ph.w[0];
  if (v1 >= ph.n_per) { v1 -= ph.n_per; b1 = ph.w[1]; if (v1 >= ph.n_per) { v1 -= ph.n_per; b1 = ph.w[2]; } }
  r.w0 = (const char*)b0 + (size_t)v0 * rowb;
  r.w1 = (const char*)b1 + (size_t)v1 * rowb;
  return r;
}

// per-task values the epilogue needs, requested with the task's first chunk
struct TaskAux {
  float b0, b1;  // bias (BIAS_*) or rotary (cos, sin) (QKV)
};

template <typename WT>
__device__ __forceinline__ void load_chunk(const TaskRows& r, int K, int c, int lane, Chunk& ch) {
  const WT* w0 = reinterpret_cast<const WT*>(r.w0);
  const WT* w1 = reinterpret_cast<const WT*>(r.w1);
  if constexpr (sizeof(WT) == 2) {
#pragma unroll
    for (int pc = 0; pc < 4; ++pc) {
      int e = c * 2048 + pc * 512 + lane * 8;
      e = e < K ? e : 0;  // past K the staged input is zero
      ch.r0[pc] = *reinterpret_cast<const uint4*>(w0 + e);
      ch.r1[pc] = *reinterpret_cast<const uint4*>(w1 + e);
    }
  } else {
#pragma unroll
    for (int pc = 0; pc < 2; ++pc) {
      int e = c * 1024 + pc * 512 + lane * 8;
      e = e < K ? e : 0;
      ch.r0[2 * pc] = *reinterpret_cast<const uint4*>(w0 + e);
      ch.r0[2 * pc + 1] = *reinterpret_cast<const uint4*>(w0 + e + 4);
      ch.r1[2 * pc] = *reinterpret_cast<const uint4*>(w1 + e);
      ch.r1[2 * pc + 1] = *reinterpret_cast<const uint4*>(w1 + e + 4);
    }
  }
}

template <typename WT>
__device__ __forceinline__ void dot_chunk(const Chunk& ch, const float* xs, int c, int lane,
                                          float& a0, float& a1) {
  constexpr int NPC = sizeof(WT) == 2 ? 4 : 2;
#pragma unroll
  for (int pc = 0; pc < NPC; ++pc) {
    const int g = c * (NPC * 64) + pc * 64 + lane;
    float x[8], w0[8], w1[8];
    xs_get8(xs, g, x);
    if constexpr (sizeof(WT) == 2) {
      unpack_bf16x8(ch.r0[pc], w0);
      unpack_bf16x8(ch.r1[pc], w1);
    } else {
      const uint4 p0 = ch.r0[2 * pc], p1 = ch.r0[2 * pc + 1];
      const uint4 q0 = ch.r1[2 * pc], q1 = ch.r1[2 * pc + 1];
      w0[0] = __uint_as_float(p0.x); w0[1] = __uint_as_float(p0.y); w0[2] = __uint_as_float(p0.z); w0[3] = __uint_as_float(p0.w);
      w0[4] = __uint_as_float(p1.x); w0[5] = __uint_as_float(p1.y); w0[6] = __uint_as_float(p1.z); w0[7] = __uint_as_float(p1.w);
      w1[0] = __uint_as_float(q0.x); w1[1] = __uint_as_float(q0.y); w1[2] = __uint_as_float(q0.z); w1[3] = __uint_as_float(q0.w);
      w1[4] = __uint_as_float(q1.x); w1[5] = __uint_as_float(q1.y); w1[6] = __uint_as_float(q1.z); w1[7] = __uint_as_float(q1.w);
    }
    float t0 = a0, t1 = a1;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      t0 = fmaf(w0[e], x[e], t0);
      t1 = fmaf(w1[e], x[e], t1);
    }
    a0 = t0;
    a1 = t1;
  }
}

__device__ __forceinline__ TaskAux load_aux(const StepPhase& ph, const StepArgs& a,
                                            const TaskRows& r, int pos) {
  TaskAux x = {0.f, 0.f};
  if (ph.epi == EPI_BIAS_GELU || ph.epi == EPI_BIAS_RESID) {
    x.b0 = ph.bias[r.n0];
    x.b1 = r.ok1 ? ph.bias[r.n1] : 0.f;
  } else if (ph.epi == EPI_QKV && r.mat < 2 && a.rope_cos) {
    const int half = a.d_head >> 1;
    const int i = r.c0 % a.d_head;
    const int tp = pos < 0 ? 0 : (pos >= a.max_seq ? a.max_seq - 1 : pos);
    x.b0 = a.rope_cos[(size_t)tp * half + i];
    x.b1 = a.rope_sin[(size_t)tp * half + i];
  }
  return x;
}

// Epilogue of one task (every lane holds r0 and r1; lane 0 stores).
template <typename KT>
__device__ __forceinline__ void finish_task(const StepPhase& ph, const StepArgs& a,
                                            const TaskRows& r, const TaskAux& aux, float r0,
                                            float r1, const float* xres, int lane, int pos,
                                            int page, float& best_v, int& best_i) {
  const int epi = ph.epi;
  if (epi == EPI_ARGMAX) {
    argmax_merge(best_v, best_i, r0, r.n0);
    if (r.ok1) argmax_merge(best_v, best_i, r1, r.n1);
    if (a.logits && lane == 0) {
      a.logits[r.n0] = r0;
      if (r.ok1) a.logits[r.n1] = r1;
    }
    return;
  }
  if (lane != 0) return;
  if (epi == EPI_QKV) {
    float e0 = r0, e1 = r1;
    const int half = a.d_head >> 1;
    if (r.mat < 2 && a.rope_cos) {
      const float c = aux.b0, s = aux.b1;
      const float t0 = e0 * c - e1 * s, t1 = e1 * c + e0 * s;
      e0 = t0;
      e1 = t1;
    }
    if (r.mat == 0) {
      st_coh(ph.y + r.c0, e0);
      st_coh(ph.y + r.c0 + half, e1);
      return;
    }
    const int pg_i = pos >= 0 ? pos / a.page_size : 0;
    if (pos < 0 || pos >= a.max_seq || pg_i >= a.max_pages) {
      atomicOr(a.status, SSD_DEV_CAPACITY);
      return;
    }
    if (page < 0 || page >= a.n_pages) {
      atomicOr(a.status, SSD_DEV_BAD_PAGE);
      return;
    }
    const int h = r.c0 / a.d_head, i = r.c0 - h * a.d_head;
    const int slot = pos - pg_i * a.page_size;
    KT* base = reinterpret_cast<KT*>(r.mat == 1 ? a.k_pool : a.v_pool) +
               (size_t)ph.layer * a.layer_elems +
               (((size_t)page * a.n_heads + h) * a.page_size + slot) * a.d_head;
    st_coh(base + i, e0);
    st_coh(base + i + half, e1);
    return;
  }
  if (epi == EPI_GATED_GELU || epi == EPI_GATED_SILU) {
    st_coh(ph.y + r.n0, (epi == EPI_GATED_GELU ? gelu_tanh(r0) : silu(r0)) * r1);
    return;
  }
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    if (s == 1 && !r.ok1) break;
    const int n = s ? r.n1 : r.n0;
    const float v = s ? r1 : r0;
    float out = v;
    if (epi == EPI_RESID) {
      out = xres[n] + v;
      if (ph.to_stash) a.stash[n] = out;
    } else if (epi == EPI_BIAS_GELU) {
      out = gelu_tanh(v + (s ? aux.b1 : aux.b0));
    } else if (epi == EPI_BIAS_RESID) {
      out = (ph.bias_resid ? xres[n] : 0.f) + (v + (s ? aux.b1 : aux.b0));
    }
    st_coh(ph.y + n, out);
  }
}

// ---------------------------------------------------------------------------------------------
// Attention of the row's query (position pos) for one (head, key split): keys
// [s * KS, min(pos + 1, (s + 1) * KS)), 16 keys per pass with 4 lanes per key (dh / 4 elements
// each); all key and value loads of the split are issued at once (at most 8 + 8 16-byte loads
// per lane).  Writes (sum_j p_j v_j, max, sum_j p_j) with p_j = exp(score_j - max).

template <typename KT, int DH>
__device__ void attn_task(const StepPhase& ph, const StepArgs& a, int t, int lane, int pos) {
  constexpr int SL = DH / 4;            // elements per lane
  constexpr int EPV = 16 / sizeof(KT);  // elements per 16-byte load
  constexpr int NV = SL / EPV;          // 16-byte loads per lane per key row
  constexpr int NP = step_attn_passes(DH, sizeof(KT));  // passes of 16 keys
  constexpr int KS = 16 * NP;
  const int S = ph.n_splits;
  const int h = t / S, s = t - h * S;
  const int g = lane >> 2, sub = lane & 3;
  const int ctx = pos + 1;
  const int k0 = s * KS;
  float* rec = ph.part + ((size_t)h * S + s) * (DH + REC);
  if (k0 >= ctx) {
    if (g == 0) {
      for (int e = 0; e < SL; e += 4) st_coh4(rec + sub * SL + e, 0.f, 0.f, 0.f, 0.f);
      if (lane == 0) {
        st_coh(rec + DH, -INFINITY);
        st_coh(rec + DH + 1, 0.f);
      }
    }
    return;
  }
  const KT* Kb = reinterpret_cast<const KT*>(a.k_pool) + (size_t)ph.layer * a.layer_elems;
  const KT* Vb = reinterpret_cast<const KT*>(a.v_pool) + (size_t)ph.layer * a.layer_elems;
  uint4 kr[NP][NV], vr[NP][NV];
  bool ok[NP];
  float bias[NP];
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    const int j = k0 + p * 16 + g;
    const int pg_i = j / a.page_size;
    int page = -1;
    if (j < ctx && pg_i < a.max_pages) page = a.page_table[pg_i];
    ok[p] = j < ctx && page >= 0 && page < a.n_pages;
    const size_t off = ok[p] ? (((size_t)page * a.n_heads + h) * a.page_size + (j - pg_i * a.page_size)) * DH + sub * SL : 0;
#pragma unroll
    for (int u = 0; u < NV; ++u) {
      kr[p][u] = *reinterpret_cast<const uint4*>(Kb + off + u * EPV);
      vr[p][u] = *reinterpret_cast<const uint4*>(Vb + off + u * EPV);
    }
    bias[p] = 0.f;
    if (a.bias_tab && ok[p] && pos - j < a.max_seq) bias[p] = a.bias_tab[(size_t)h * a.max_seq + (pos - j)];
  }
  float qv[SL];
#pragma unroll
  for (int e = 0; e < SL; e += 4) {
    const float4 q4 = *reinterpret_cast<const float4*>(ph.q + h * DH + sub * SL + e);
    qv[e] = q4.x * a.attn_scale; qv[e + 1] = q4.y * a.attn_scale;
    qv[e + 2] = q4.z * a.attn_scale; qv[e + 3] = q4.w * a.attn_scale;
  }
  float sc[NP];
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    float d = 0.f;
#pragma unroll
    for (int u = 0; u < NV; ++u) {
      float kf[EPV];
      if constexpr (sizeof(KT) == 2) {
        unpack_bf16x8(kr[p][u], kf);
      } else {
        kf[0] = __uint_as_float(kr[p][u].x); kf[1] = __uint_as_float(kr[p][u].y);
        kf[2] = __uint_as_float(kr[p][u].z); kf[3] = __uint_as_float(kr[p][u].w);
      }
#pragma unroll
      for (int e = 0; e < EPV; ++e) d = fmaf(qv[u * EPV + e], kf[e], d);
    }
    d += __shfl_xor(d, 1, 64);
    d += __shfl_xor(d, 2, 64);
    sc[p] = ok[p] ? d + bias[p] : -INFINITY;
  }
  float m = sc[0];
#pragma unroll
  for (int p = 1; p < NP; ++p) m = fmaxf(m, sc[p]);
  m = wave_max(m);
  float pr[NP], lsum = 0.f;
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    pr[p] = ok[p] ? __expf(sc[p] - m) : 0.f;
    lsum += sub == 0 ? pr[p] : 0.f;
  }
  lsum = wave_sum(lsum);
  float o[SL];
#pragma unroll
  for (int e = 0; e < SL; ++e) o[e] = 0.f;
#pragma unroll
  for (int p = 0; p < NP; ++p) {
#pragma unroll
    for (int u = 0; u < NV; ++u) {
      float vf[EPV];
      if constexpr (sizeof(KT) == 2) {
        unpack_bf16x8(vr[p][u], vf);
      } else {
        vf[0] = __uint_as_float(vr[p][u].x); vf[1] = __uint_as_float(vr[p][u].y);
        vf[2] = __uint_as_float(vr[p][u].z); vf[3] = __uint_as_float(vr[p][u].w);
      }
#pragma unroll
      for (int e = 0; e < EPV; ++e) o[u * EPV + e] = fmaf(pr[p], vf[e], o[u * EPV + e]);
    }
  }
  // sum over the 16 keys of a pass (lanes with equal sub)
#pragma unroll
  for (int e = 0; e < SL; ++e) {
    float v = o[e];
    v += __shfl_xor(v, 4, 64);
    v += __shfl_xor(v, 8, 64);
    v += __shfl_xor(v, 16, 64);
    v += __shfl_xor(v, 32, 64);
    o[e] = v;
  }
  if (g == 0) {
#pragma unroll
    for (int e = 0; e < SL; e += 4) st_coh4(rec + sub * SL + e, o[e], o[e + 1], o[e + 2], o[e + 3]);
    if (lane == 0) {
      st_coh(rec + DH, m);
      st_coh(rec + DH + 1, lsum);
    }
  }
}

// Merge of the key-split partials of one head into its dh outputs (one wave per head).
__device__ void combine_task(const StepPhase& ph, int h, int lane, int dh) {
  const int S = ph.n_splits;
  const float* rec = ph.part + (size_t)h * S * (dh + REC);
  float mx = lane < S ? rec[(size_t)lane * (dh + REC) + dh] : -INFINITY;
  float ls = lane < S ? rec[(size_t)lane * (dh + REC) + dh + 1] : 0.f;
  const float M = wave_max(mx);
  const float w = (lane < S && mx != -INFINITY) ? __expf(mx - M) : 0.f;
  const float L = wave_sum(w * ls);
  const float inv = 1.0f / L;
  for (int e = lane; e < dh; e += 64) {
    float acc = 0.f;
    for (int s = 0; s < S; ++s) acc = fmaf(__shfl(w, s, 64), rec[(size_t)s * (dh + REC) + e], acc);
    st_coh(ph.y + h * dh + e, acc * inv);
  }
}

// ---------------------------------------------------------------------------------------------

template <typename KT>
__global__ __launch_bounds__(ST_THREADS) void step_kernel(const StepArgs a) {
  __shared__ __attribute__((aligned(16))) float xs[STEP_XS_MAX];
  __shared__ __attribute__((aligned(16))) float xres[STEP_XRES_MAX];
  __shared__ float rv[ST_WAVES];
  __shared__ int ri[ST_WAVES];
  __shared__ float nscale;
  __shared__ int go, last;
  __shared__ uint32_t base_s;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int nblk = gridDim.x, blk = blockIdx.x;
  if (tid == 0) {
    base_s = ld_coh(a.flags + blk);
    const bool ab = ld_coh(a.abort_word) != 0u;
    go = ab ? 0 : 1;
    if (ab && blk == 0) atomicOr(a.status, SSD_DEV_SYNC);
  }
  __syncthreads();
  if (!go) return;
  const uint32_t base = base_s;
  const int pos = a.seq_len[0] + a.pos_off;
  // the page that holds this row's K / V (an out-of-range position is reported at the store)
  const int pos_pg = pos >= 0 ? pos / a.page_size : 0;
  const int kv_page = a.page_table[pos_pg < a.max_pages ? pos_pg : a.max_pages - 1];
  const int gw = wave * nblk + blk;  // this compute wave's index over the grid
  const int W = ST_CW * nblk;
  const bool compute = wave < ST_CW;

  for (int p = 0; p < a.n_phases; ++p) {
    const StepPhase& ph = a.phases[p];
    const int type = ph.type;
    const bool gemv = type == SP_GEMV;
    const int f32w = ph.wdtype == SSD_F32;
    const int esz = f32w ? 4 : 2;
    const int nt = ph.n_tasks;
    const int K = ph.K;
    const int CE = f32w ? 1024 : 2048;
    const int nc = (K + CE - 1) / CE;

    // request the weights of the first task before the barrier
    int t = gw;
    TaskRows rows = {};
    TaskAux aux = {0.f, 0.f};
    Chunk cur;
    if (gemv && compute && t < nt) {
      rows = task_rows(ph, t, esz, a.d_head);
      if (f32w) load_chunk<float>(rows, K, 0, lane, cur);
      else load_chunk<bf16_t>(rows, K, 0, lane, cur);
      aux = load_aux(ph, a, rows, pos);
    }

    // barrier: every block has finished phase p - 1
    if (p > 0) {
      if (wave == ST_CW) {
        const bool ok = poll_flags(a, base + (uint32_t)p, lane, nblk);
        if (lane == 0) go = ok ? 1 : 0;
      }
      __syncthreads();
      if (!go) return;
    }

    if (gemv) {
      // stage the input row
      if (ph.in_kind == SI_ATTN) {
        stage_attn(ph, xs, tid, a.d_head);
        if (tid == 0) nscale = 1.f;
      } else if (wave == ST_CW) {
        if (ph.in_kind == SI_EMBED) {
          int tok = a.tok[0];
          if (tok < 0 || tok >= a.vocab) {
            if (lane == 0 && blk == 0) atomicOr(a.status, SSD_DEV_BAD_TOKEN);
            tok = 0;
          }
          if (a.wdtype == SSD_F32)
            stage_row<float>(ph, reinterpret_cast<const float*>(a.embed) + (size_t)tok * a.d_model,
                             xs, xres, &nscale, lane);
          else
            stage_row<bf16_t>(ph, reinterpret_cast<const bf16_t*>(a.embed) + (size_t)tok * a.d_model,
                              xs, xres, &nscale, lane);
        } else {
          stage_row<float>(ph, ph.x, xs, xres, &nscale, lane);
        }
      }
      __syncthreads();

      float best_v = -INFINITY;
      int best_i = INT_MAX;
      if (compute && t < nt) {
        const float sc = nscale;
        float a0 = 0.f, a1 = 0.f;
        int c = 0;
        while (true) {
          int t2 = t, c2 = c + 1;
          if (c2 == nc) {
            c2 = 0;
            t2 = t + W;
          }
          Chunk nxt;
          TaskRows rows2 = rows;
          TaskAux aux2 = aux;
          if (t2 < nt) {
            if (c2 == 0) rows2 = task_rows(ph, t2, esz, a.d_head);
            if (f32w) load_chunk<float>(rows2, K, c2, lane, nxt);
            else load_chunk<bf16_t>(rows2, K, c2, lane, nxt);
            if (c2 == 0) aux2 = load_aux(ph, a, rows2, pos);
          }
          if (f32w) dot_chunk<float>(cur, xs, c, lane, a0, a1);
          else dot_chunk<bf16_t>(cur, xs, c, lane, a0, a1);
          if (c == nc - 1) {
            // rows n0 (lanes 0..31 after the first exchange) and n1 (lanes 32..63)
            const bool hi = lane & 32;
            float u = hi ? a1 : a0;
            const float v = hi ? a0 : a1;
            u += __shfl_xor(v, 32, 64);
            u += __shfl_xor(u, 16, 64);
            u += __shfl_xor(u, 8, 64);
            u += __shfl_xor(u, 4, 64);
            u += __shfl_xor(u, 2, 64);
            u += __shfl_xor(u, 1, 64);
            const float r0 = __shfl(u, 0, 64) * sc, r1 = __shfl(u, 32, 64) * sc;
            finish_task<KT>(ph, a, rows, aux, r0, r1, xres, lane, pos, kv_page, best_v, best_i);
            a0 = a1 = 0.f;
          }
          if (t2 >= nt) break;
          cur = nxt;
          rows = rows2;
          aux = aux2;
          t = t2;
          c = c2;
        }
      }

      if (ph.epi == EPI_ARGMAX) {
        // block's best -> one partial per block; the last block to arrive reduces them
        if (lane == 0) {
          rv[wave] = best_v;
          ri[wave] = best_i;
        }
        __syncthreads();
        if (tid == 0) {
          float v = rv[0];
          int i = ri[0];
          for (int w = 1; w < ST_WAVES; ++w) argmax_merge(v, i, rv[w], ri[w]);
          st_coh(a.part_val + blk, v);
          st_coh(a.part_idx + blk, i);
          __builtin_amdgcn_s_waitcnt(0);
          const uint32_t old = __hip_atomic_fetch_add(a.counter, 1u, __ATOMIC_RELAXED,
                                                       __HIP_MEMORY_SCOPE_AGENT);
          last = old == (uint32_t)(nblk - 1) ? 1 : 0;
        }
        __syncthreads();
        if (last && wave == 0) {
          float v = -INFINITY;
          int i = INT_MAX;
          for (int b = lane; b < nblk; b += 64) argmax_merge(v, i, a.part_val[b], a.part_idx[b]);
          wave_argmax(v, i);
          if (lane == 0) {
            if (i == INT_MAX) i = 0;  // every logit NaN: nothing sensible to choose
            a.dst0[0] = i;
            if (a.dst1) a.dst1[0] = i;
            st_coh(a.counter, 0u);
          }
        }
      }
    } else {
      if (compute) {
        for (int tt = gw; tt < nt; tt += W) {
          if (type == SP_ATTN) {
            if (a.d_head == 64) attn_task<KT, 64>(ph, a, tt, lane, pos);
            else attn_task<KT, 128>(ph, a, tt, lane, pos);
          } else {
            combine_task(ph, tt, lane, a.d_head);
          }
        }
      }
    }

    // publish: this block's outputs of phase p are complete
    if (p + 1 < a.n_phases) {
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
      if (tid == 0) st_coh(a.flags + blk, base + (uint32_t)p + 1u);
    }
  }
}

int g_step_blocks = -1;

}  // namespace

int step_blocks() {
  if (g_step_blocks >= 0) return g_step_blocks;
  int dev = 0, cus = 0, occ = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, step_kernel<float>, ST_THREADS, 0) !=
          hipSuccess) {
    g_step_blocks = 0;
    return 0;
  }
  int occ2 = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ2, step_kernel<bf16_t>, ST_THREADS, 0) !=
      hipSuccess)
    occ2 = 0;
  const bool ok = occ >= 1 && occ2 >= 1 && cus >= 1 && cus <= STEP_MAX_BLOCKS;
  g_step_blocks = ok ? cus : 0;
  return g_step_blocks;
}

hipError_t launch_step(const StepArgs& a, int kvdtype, hipStream_t s, hipEvent_t start,
                       hipEvent_t stop) {
  const int nb = step_blocks();
  if (nb <= 0) return hipErrorInvalidConfiguration;
  if (start && stop) {
    if (kvdtype == SSD_BF16)
      hipExtLaunchKernelGGL(step_kernel<bf16_t>, dim3(nb), dim3(ST_THREADS), 0, s, start, stop, 0, a);
    else
      hipExtLaunchKernelGGL(step_kernel<float>, dim3(nb), dim3(ST_THREADS), 0, s, start, stop, 0, a);
  } else {
    if (kvdtype == SSD_BF16)
      hipLaunchKernelGGL(step_kernel<bf16_t>, dim3(nb), dim3(ST_THREADS), 0, s, a);
    else
      hipLaunchKernelGGL(step_kernel<float>, dim3(nb), dim3(ST_THREADS), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace ssd
