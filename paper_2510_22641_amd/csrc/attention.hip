// Softmax attention of a block of query rows of one head.
//
// Self-attention: query row j of sequence b sits at position p = seq_len[b] + pos_off + j and
// attends keys 0..p of the paged cache (causal inside a verify chunk or a prefill block), with the
// T5 relative-position bias bias[h][p - i] added (no scaling; T5 folds it into the weights) or,
// for LLaMA, scaled by 1/sqrt(dh) with q and k already rotated.  Cross-attention (T5): all n_keys
// visual keys, no mask, no bias, no scale.
//
// One block per (head, sequence, query row) for single rows and short-context chunks of up to 16
// rows, else per (head, sequence, 8 query rows); long contexts split each head's keys over several
// blocks whose partials attn_combine_kernel merges.  Every thread issues its key row and its
// first value chunks before the first barrier (they do not depend on the scores); scores for the
// live rows go to LDS, one wave per row turns them into softmax numerators, and P.V splits the
// keys over all threads (16-byte value chunks, 8 loads in flight per thread) with a shuffle + LDS
// reduction.  Bound: bytes of K and V read (HBM/L2) and one or two memory round trips.
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

// Page-table entry of key i of sequence b (clamped to the table; validated where it is used).
__device__ __forceinline__ int key_page(const AttnArgs& a, int b, int i) {
  const int pg_i = min(i / a.kv.page_size, a.kv.max_pages - 1);
  return a.kv.page_table[(size_t)b * a.kv.max_pages + pg_i];
}

// key_row for a page-table entry already loaded.
template <typename KT, int DH>
__device__ __forceinline__ const KT* key_row_at(const AttnArgs& a, const KT* base, int h, int i,
                                                int page, bool& ok) {
  ok = i / a.kv.page_size < a.kv.max_pages && page >= 0 && page < a.kv.n_pages;
  if (!ok) page = 0;
  const int slot = i - (i / a.kv.page_size) * a.kv.page_size;
  return base + (((size_t)page * a.H + h) * a.kv.page_size + slot) * DH;
}

// Buffer-resource loads of key / value rows: 32-bit byte offsets from a pool base, and an offset
// past the resource's range (ATTN_OOB) returns zeros without a memory access, so masked lanes
// need no branch and cost no traffic.
typedef uint32_t attn_u32x4 __attribute__((ext_vector_type(4)));
constexpr uint32_t ATTN_OOB = 0x80000000u;
constexpr size_t ATTN_RS_MAX = 0x7fff0000u;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t attn_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), 0, (int)bytes, 0x00020000);
}

// Bytes of the key (or value) pool a launch may read from its base.
template <typename KT, int DH>
__host__ __device__ size_t attn_pool_bytes(const AttnArgs& a) {
  const size_t row = (size_t)DH * sizeof(KT);
  return a.cross ? (size_t)a.B * a.H * a.n_keys * row
                 : (size_t)a.kv.n_pages * a.H * a.kv.page_size * row;
}
__device__ __forceinline__ void load_rs(Vec8<bf16_t>& v, __amdgpu_buffer_rsrc_t r, uint32_t off) {
  const attn_u32x4 t = __builtin_bit_cast(attn_u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
  v.r = make_uint4(t.x, t.y, t.z, t.w);
}
__device__ __forceinline__ void load_rs(Vec8<float>& v, __amdgpu_buffer_rsrc_t r, uint32_t off) {
  const attn_u32x4 t0 = __builtin_bit_cast(attn_u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
  const attn_u32x4 t1 =
      __builtin_bit_cast(attn_u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off + 16u, 0, 0));
  v.a = make_float4(__uint_as_float(t0.x), __uint_as_float(t0.y), __uint_as_float(t0.z), __uint_as_float(t0.w));
  v.b = make_float4(__uint_as_float(t1.x), __uint_as_float(t1.y), __uint_as_float(t1.z), __uint_as_float(t1.w));
}

// RS: the layer's key and value pools span less than 2 GiB and are read with buffer loads.
template <typename KT, int DH, int QB, bool RS>
__global__ __launch_bounds__(256) void attn_kernel(const AttnArgs a, const int s_stride, const int ks) {
  constexpr int CH = DH / 8;       // 16-byte chunks per key row (bf16) / 8-element groups
  constexpr int KPI = 256 / CH;    // keys per block step in P.V
  constexpr int KPW = 64 / CH;     // keys per wave step in P.V
  constexpr int PF = 8;            // P.V loads in flight per thread
  extern __shared__ float S[];     // [QB][s_stride] scores, then unnormalised probabilities
  __shared__ float qs[QB][DH];
  __shared__ float red[4][QB][DH];
  __shared__ float inv_sum[QB];
  __shared__ float row_max[QB], row_sum[QB];

  // blockIdx.z = query group * ks + key split: this block's keys are [k0, k0 + nk) of the group's
  // causal range (ks = 1: all of them)
  const int h = blockIdx.x, b = blockIdx.y;
  const int zq = blockIdx.z / ks, split = blockIdx.z - zq * ks, j0 = zq * QB;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nq = min(QB, a.C - j0);
  const int HD = a.H * DH;
  // Every load of the prologue is issued on every path (a masked lane reads zeros or a valid
  // row, never skips the load): the wait counter retires loads in issue order, and a load skipped
  // on one path makes the compiler wait for everything issued before the next one.
  // The query rows first (they depend on nothing), then the page-table entries, the sequence
  // length, the key row, the value chunks and the position bias.
  constexpr int QPT = (QB * DH + 255) / 256;  // query elements per thread
  float qv[QPT];
#pragma unroll
  for (int t = 0; t < QPT; ++t) {
    const int idx = min(tid + 256 * t, QB * DH - 1);
    const int jq = min(idx / DH, nq - 1), d = idx - (idx / DH) * DH;
    qv[t] = a.q[(size_t)(b * a.C + j0 + jq) * HD + h * DH + d];
  }
  // the sequence length as a vector load issued now (a scalar load would be issued where it is
  // first used, after the key and value loads, and the bias would wait for it); cross-attention
  // reads a placeholder
  int vzero;
  asm volatile("v_mov_b32 %0, 0" : "=v"(vzero));
  const int* slp = a.cross ? reinterpret_cast<const int*>(a.q) : a.kv.seq_len + b;
  const int seq_len_v = slp[vzero];
  // self-attention key ranges do not depend on the sequence length (one split: from 0; several:
  // fixed ranges of ceil(max_seq / ks) keys, the last ones empty while the context is short), so
  // the page-table entries of this thread's first key row and value chunks are requested
  // together with the sequence length, not after it
  const bool pre = !a.cross;
  const int kfix = ks == 1 ? 0 : (a.max_seq + ks - 1) / ks, kbase = split * kfix;
  constexpr int PF0 = 8;  // value chunks prefetched per thread (PF below)
  const int vk00 = tid / (DH / 8), kpi0 = 256 / (DH / 8);
  int kpg = 0, vpg[PF0];
  if (pre) {
    kpg = key_page(a, b, kbase + tid);
#pragma unroll
    for (int u = 0; u < PF0; ++u) vpg[u] = key_page(a, b, kbase + vk00 + kpi0 * u);
  }
  const KT* Kb = reinterpret_cast<const KT*>(a.cross ? a.xk : a.kv.k);
  const KT* Vb = reinterpret_cast<const KT*>(a.cross ? a.xv : a.kv.v);

  const int base = a.cross ? 0 : __builtin_amdgcn_readfirstlane(seq_len_v) + a.kv.pos_off;
  const int nk_all = a.cross ? a.n_keys : base + j0 + nq;
  const int per = ks == 1 ? nk_all : kfix;
  const int k0 = min(nk_all, split * per);
  int nk = min(nk_all, k0 + per) - k0;
  if (nk > s_stride) {
    if (tid == 0) atomicOr(a.status, SSD_DEV_CAPACITY);
    nk = s_stride;
  }

  // the first key row and the first value chunks, before any barrier.  Self-attention addresses
  // them from the split's fixed start (a non-empty split starts there) and the page-table
  // entries.  Lanes past nk (and rows of a missing page) are masked: buffer loads with an
  // out-of-range offset (RS), else a clamped valid row.
  const int clast = a.n_keys - 1;
  const uint32_t pool_rs = RS ? (uint32_t)attn_pool_bytes<KT, DH>(a) : 0u;
  const __amdgpu_buffer_rsrc_t krs = attn_rsrc(Kb, pool_rs), vrs = attn_rsrc(Vb, pool_rs);
  bool kok = false;
  Vec8<KT> krow[CH];
  {
    const KT* kp = pre ? key_row_at<KT, DH>(a, Kb, h, kbase + tid, kpg, kok)
                       : key_row<KT, DH>(a, Kb, b, h, min(tid, clast), kok);
    kok = kok && tid < nk;
    if constexpr (RS) {
      const uint32_t off = kok ? (uint32_t)((size_t)(kp - Kb) * sizeof(KT)) : ATTN_OOB;
#pragma unroll
      for (int c = 0; c < CH; ++c) load_rs(krow[c], krs, off + 8u * c * sizeof(KT));
    } else {
#pragma unroll
      for (int c = 0; c < CH; ++c) krow[c].load(kp + 8 * c);
    }
  }
  const int vc = tid % CH, vk0 = tid / CH;
  static_assert(PF == PF0, "value prefetch depth");
  Vec8<KT> vpre[PF];
  bool vok[PF];
#pragma unroll
  for (int u = 0; u < PF; ++u) {
    const int i = vk0 + KPI * u;
    const KT* vp = pre ? key_row_at<KT, DH>(a, Vb, h, kbase + i, vpg[u], vok[u])
                       : key_row<KT, DH>(a, Vb, b, h, min(i, clast), vok[u]);
    vok[u] = vok[u] && i < nk;
    if constexpr (RS) {
      const uint32_t off = vok[u] ? (uint32_t)((size_t)(vp - Vb + 8 * vc) * sizeof(KT)) : ATTN_OOB;
      load_rs(vpre[u], vrs, off);
    } else {
      vpre[u].load(vp + 8 * vc);
    }
  }
  // T5 position bias of this thread's first key for each query row (LLaMA and cross-attention:
  // a placeholder read of the query)
  float bpre[QB];
  {
    const float* bsrc = (a.bias && !a.cross) ? a.bias + (size_t)h * a.max_seq : a.q;
#pragma unroll
    for (int jq = 0; jq < QB; ++jq) {
      const int dist = base + j0 + jq - (k0 + tid);
      bpre[jq] = bsrc[(a.bias && !a.cross) ? min(max(dist, 0), a.max_seq - 1) : 0];
    }
  }

#pragma unroll
  for (int t = 0; t < QPT; ++t) {
    const int idx = tid + 256 * t;
    if (idx < QB * DH) {
      const int jq = idx / DH, d = idx - jq * DH;
      qs[jq][d] = jq < nq ? qv[t] * a.scale : 0.f;
    }
  }
  __syncthreads();

  // scores: one key per thread per step (i relative to k0)
  for (int i = tid; i < nk; i += 256) {
    // query blocks and 512-byte key rows: the query reads stay inside the loop (hoisted out of
    // it they pin up to 8 rows of registers, and spill with float keys at dh 128); a one-row
    // block with a short key row keeps them hoisted
    if constexpr (QB > 1 || DH * sizeof(KT) > 256) asm volatile("" ::: "memory");
    bool ok = kok;
    if (i != tid) {
      const KT* kp = key_row<KT, DH>(a, Kb, b, h, k0 + i, ok);
      if (ok) {
#pragma unroll
        for (int c = 0; c < CH; ++c) krow[c].load(kp + 8 * c);
      }
    }
    float dots[QB];
#pragma unroll
    for (int jq = 0; jq < QB; ++jq) dots[jq] = 0.f;
    if (ok) {
#pragma unroll
      for (int c = 0; c < CH; ++c) {
        float kf[8];
        krow[c].to_f32(kf);
        // every row of the block (rows past nq hold zeros and are masked below): no branch
        // between the LDS reads of the rows, so they are issued together
#pragma unroll
        for (int jq = 0; jq < QB; ++jq) {
          float t = dots[jq];
#pragma unroll
          for (int e = 0; e < 8; ++e) t = fmaf(qs[jq][8 * c + e], kf[e], t);
          dots[jq] = t;
        }
      }
    }
#pragma unroll
    for (int jq = 0; jq < QB; ++jq) {
      float sc = dots[jq];
      if (!ok || jq >= nq) {
        sc = -INFINITY;
      } else if (!a.cross) {
        const int p = base + j0 + jq, ki = k0 + i;
        if (ki > p) sc = -INFINITY;
        else if (a.bias && p - ki < a.max_seq)
          sc += i == tid ? bpre[jq] : a.bias[(size_t)h * a.max_seq + (p - ki)];
      }
      S[jq * s_stride + i] = sc;
    }
  }
  __syncthreads();

  // softmax numerators, one wave per row
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
    if (lane == 0) {
      inv_sum[jq] = sum > 0.f ? 1.0f / sum : 0.f;
      row_max[jq] = m;
      row_sum[jq] = sum;
    }
  }
  __syncthreads();

  // P . V: thread (key group vk0, chunk vc) accumulates 8 dims of every query row
  float acc[QB][8];
#pragma unroll
  for (int jq = 0; jq < QB; ++jq)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[jq][e] = 0.f;
  for (int u0 = 0; vk0 + KPI * u0 < nk; u0 += PF) {
    if (u0 > 0) {
#pragma unroll
      for (int u = 0; u < PF; ++u) {
        const int i = vk0 + KPI * (u0 + u);
        vok[u] = false;
        if (i < nk) {
          const KT* vp = key_row<KT, DH>(a, Vb, b, h, k0 + i, vok[u]);
          if (vok[u]) vpre[u].load(vp + 8 * vc);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < PF; ++u) {
      const int i = vk0 + KPI * (u0 + u);
      if (i < nk && vok[u]) {
        float vf[8];
        vpre[u].to_f32(vf);
#pragma unroll
        for (int jq = 0; jq < QB; ++jq) {
          // rows past nq (scores never turned into probabilities) contribute nothing
          const float sp = S[jq * s_stride + i];
          const float p = jq < nq ? sp : 0.f;
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[jq][e] = fmaf(p, vf[e], acc[jq][e]);
        }
      }
    }
  }
  // reduce over the key groups of the wave (lanes that share vc), then over waves
#pragma unroll
  for (int jq = 0; jq < QB; ++jq)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      float v = acc[jq][e];
#pragma unroll
      for (int o = CH; o < 64; o <<= 1) v += __shfl_xor(v, o, SSD_WAVE);
      acc[jq][e] = v;
    }
  if (lane < CH) {
#pragma unroll
    for (int jq = 0; jq < QB; ++jq)
#pragma unroll
      for (int e = 0; e < 8; ++e) red[wave][jq][8 * lane + e] = acc[jq][e];
  }
  __syncthreads();
  for (int idx = tid; idx < nq * DH; idx += 256) {
    const int jq = idx / DH, d = idx - jq * DH;
    const float v = (red[0][jq][d] + red[1][jq][d]) + (red[2][jq][d] + red[3][jq][d]);
    if (ks > 1) {
      // partial of this key split: unnormalised output, row max and sum (attn_combine_kernel)
      float* pp = a.part + (((size_t)(b * a.C + j0 + jq) * a.H + h) * ks + split) * (DH + 2);
      pp[d] = v;
      if (d == 0) {
        pp[DH] = row_max[jq];
        pp[DH + 1] = row_sum[jq];
      }
      continue;
    }
    const size_t o = (size_t)(b * a.C + j0 + jq) * HD + h * DH + d;
    a.out[o] = v * inv_sum[jq];
    if (a.out_planes) {  // hi / lo bf16 planes for the skinny MFMA consumer (rows < plane_rows)
      const float y = v * inv_sum[jq];
      const uint32_t hi = f32_to_bf16(y);
      a.out_planes[o] = (bf16_t)hi;
      a.out_planes[o + (size_t)a.plane_rows * HD] = (bf16_t)f32_to_bf16(y - bf16_to_f32(hi));
    }
  }
}

// Merge the key splits of one (head, row): out = sum_s e^(m_s - m) o_s / sum_s e^(m_s - m) l_s.
template <int DH>
__global__ __launch_bounds__(DH) void attn_combine_kernel(const AttnArgs a, const int ks) {
  const int h = blockIdx.x, r = blockIdx.y, d = threadIdx.x;
  const int HD = a.H * DH;
  const float* pp = a.part + ((size_t)r * a.H + h) * ks * (DH + 2);
  // every split's max, sum and output requested before the first is used (one memory round trip
  // instead of one per split); indexes past ks re-read the last split and are not used
  float ms[ATTN_SPLITS_MAX], ls[ATTN_SPLITS_MAX], os[ATTN_SPLITS_MAX];
#pragma unroll
  for (int sp = 0; sp < ATTN_SPLITS_MAX; ++sp) {
    const float* q = pp + (size_t)min(sp, ks - 1) * (DH + 2);
    ms[sp] = q[DH];
    ls[sp] = q[DH + 1];
    os[sp] = q[d];
  }
  float m = -INFINITY;
#pragma unroll
  for (int sp = 0; sp < ATTN_SPLITS_MAX; ++sp)
    if (sp < ks) m = fmaxf(m, ms[sp]);
  float l = 0.f, o = 0.f;
#pragma unroll
  for (int sp = 0; sp < ATTN_SPLITS_MAX; ++sp)
    if (sp < ks) {
      const float w = ms[sp] == -INFINITY ? 0.f : expf(ms[sp] - m);
      l = fmaf(w, ls[sp], l);
      o = fmaf(w, os[sp], o);
    }
  const float y = l > 0.f ? o / l : 0.f;
  const size_t oi = (size_t)r * HD + h * DH + d;
  a.out[oi] = y;
  if (a.out_planes) {
    const uint32_t hi = f32_to_bf16(y);
    a.out_planes[oi] = (bf16_t)hi;
    a.out_planes[oi + (size_t)a.plane_rows * HD] = (bf16_t)f32_to_bf16(y - bf16_to_f32(hi));
  }
}

// Causal self-attention of a prefill block on MFMA (float32 cache, no position bias): one block of
// four waves per (64 query rows, head, sequence), wave w owning rows 16w..16w+15.  Keys advance in
// tiles of 64 staged in LDS as bf16 hi / lo planes (K by key row, V transposed by dimension); the
// next tile is loaded into registers while the current one is used.  Per 16-key sub-tile a wave
// computes S^T = K . Q^T with v_mfma_f32_16x16x32_bf16 (hi.hi + hi.lo + lo.hi, about 16 mantissa
// bits per operand), so lane l holds the scores of query l % 16; the online softmax (running max
// and sum per query) therefore stays in the lane, and O^T += V^T . P^T takes the lane's own
// probabilities as its B operand (the K index of the product runs over keys 4g..4g+3 of two
// sub-tiles, g = l / 16, and the V^T operand is read in the same order).  The block's 8 waves are
// two halves over the same query rows: half 0 takes the even key tiles, half 1 the odd ones, each
// with its own LDS stage, and the two running (max, sum, output) triples are merged through LDS at
// the end, which halves the longest chain of key tiles.  Blocks are issued longest (last query
// rows) first.
template <int DH>
__global__ __launch_bounds__(512) void attn_mfma_kernel(const AttnArgs a, const int n_qt) {
  constexpr int KT = 64;        // keys per tile
  constexpr int KLD = DH + 8;   // bf16 per key row of the K planes
  constexpr int VLD = KT + 4;   // bf16 per dimension row of the V^T planes (34 dwords: the
                                // transposed stores of a wave hit 64 distinct banks)
  constexpr int NC = DH / 32;   // head-dim chunks of the score products
  constexpr int ND = DH / 16;   // output dimension tiles per wave
  constexpr int KF = DH / 4;    // K floats a thread stages (4 threads per key)
  constexpr int VF = DH / 8;    // V floats per key a thread stages (8 threads per key pair)
  constexpr int STAGE = 2 * KT * KLD + 2 * DH * VLD;  // bf16 of one half's stage
  extern __shared__ __attribute__((aligned(16))) bf16_t am_s[];
  const int half = threadIdx.x >> 8;
  bf16_t* Ks = am_s + half * STAGE;    // [2][KT][KLD]  hi, lo
  bf16_t* Vt = Ks + 2 * KT * KLD;      // [2][DH][VLD]  hi, lo
  int* pg = reinterpret_cast<int*>(am_s + 2 * STAGE);  // [n_pg] page-table entries of the keys

  // (query tile, head, sequence) of this block: workgroups are dealt to the 8 XCDs round-robin
  // by linear id, so the id is mapped to a contiguous range of tiles per XCD, query tiles fastest
  // (longest first): the query tiles of a head share its keys and values in one XCD's L2
  // (longest first); when an XCD's range is whole heads, its blocks go level by level over those
  // heads, so that the blocks left for a second round on the XCD's compute units are short ones
  int qt, h, b;
  {
    const int T = n_qt * gridDim.y * gridDim.z;
    const int id = blockIdx.x + n_qt * (blockIdx.y + gridDim.y * blockIdx.z);
    const int xcd = id & 7;
    int slot = id >> 3;
    const int start = xcd * (T >> 3) + min(xcd, T & 7), cnt = (T >> 3) + (xcd < (T & 7) ? 1 : 0);
    if (start % n_qt == 0 && cnt % n_qt == 0) {
      const int nh = cnt / n_qt;
      slot = (slot % nh) * n_qt + slot / nh;
    }
    const int t = start + slot;
    qt = n_qt - 1 - t % n_qt;
    const int rest = t / n_qt;
    h = rest % gridDim.y;
    b = rest / gridDim.y;
  }
  const int tid = threadIdx.x & 255, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, c16 = lane & 15;
  const int j0 = qt * 64;
  const int nq = min(64, a.C - j0);
  const int HD = a.H * DH;
  const int base = a.kv.seq_len[b] + a.kv.pos_off;
  int nk = base + j0 + nq;
  if (nk > a.max_seq) {
    if (tid == 0) atomicOr(a.status, SSD_DEV_CAPACITY);
    nk = a.max_seq;
  }
  const int n_kt = (nk + KT - 1) / KT;
  const float* Kp = reinterpret_cast<const float*>(a.kv.k);
  const float* Vp = reinterpret_cast<const float*>(a.kv.v);
  // the page-table entries of keys 0..nk-1 in LDS once, so that a tile's loads depend on one
  // memory round trip, not two (-1: past the table)
  const int n_pg = (nk + a.kv.page_size - 1) / a.kv.page_size;
  for (int i = threadIdx.x; i < n_pg; i += 512)
    pg[i] = i < a.kv.max_pages ? a.kv.page_table[(size_t)b * a.kv.max_pages + i] : -1;
  __syncthreads();

  // staging roles: K key tid / 4, floats (tid % 4) * KF ..; V keys 2 (tid % 32) and + 1, floats
  // (tid / 32) * VF .. (a wave's transposed stores then cover 32 key pairs of two dimension
  // groups: 64 distinct banks)
  const int kk_l = tid >> 2, kd0 = (tid & 3) * KF;
  const int vp_l = tid & 31, vd0 = (tid >> 5) * VF;
  float4 kr[KF / 4], vr[2][VF / 4];
  bool kok = false, vok[2] = {false, false};
  // pages hold a power of two of keys dividing the tile: a thread's keys sit at fixed page
  // offsets and slots in every tile
  const int lps = __builtin_ctz(a.kv.page_size), ppt = KT >> lps;
  const int k_pg = kk_l >> lps, k_slot = kk_l & (a.kv.page_size - 1);
  const int v_pg = (2 * vp_l) >> lps, v_slot = (2 * vp_l) & (a.kv.page_size - 1);
  const size_t pstride = (size_t)a.H * a.kv.page_size * DH, hoff = (size_t)h * a.kv.page_size * DH;
  auto fetch = [&](int kt) {
    int page = pg[min(kt * ppt + k_pg, n_pg - 1)];
    kok = kt * KT + kk_l < nk && page >= 0 && page < a.kv.n_pages;
    const float* src = Kp + (size_t)(kok ? page : 0) * pstride + hoff + (size_t)k_slot * DH + kd0;
#pragma unroll
    for (int q = 0; q < KF / 4; ++q) kr[q] = reinterpret_cast<const float4*>(src)[q];
    page = pg[min(kt * ppt + v_pg, n_pg - 1)];
    const bool vp_ok = page >= 0 && page < a.kv.n_pages;
    const float* vs = Vp + (size_t)(vp_ok ? page : 0) * pstride + hoff + (size_t)v_slot * DH + vd0;
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      vok[u] = vp_ok && kt * KT + 2 * vp_l + u < nk;
#pragma unroll
      for (int q = 0; q < VF / 4; ++q) vr[u][q] = reinterpret_cast<const float4*>(vs + u * DH)[q];
    }
  };
  if (half < n_kt) fetch(half);

  // this wave's query rows as the B operand (hi / lo), pre-scaled; rows past nq repeat the last
  bf16x8_t qh[NC], ql[NC];
  {
    const float* qrow = a.q + (size_t)(b * a.C + j0 + min(16 * wave + c16, nq - 1)) * HD + h * DH;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const float4 u0 = reinterpret_cast<const float4*>(qrow + 32 * c + 8 * g)[0];
      const float4 u1 = reinterpret_cast<const float4*>(qrow + 32 * c + 8 * g)[1];
      float f[8] = {u0.x, u0.y, u0.z, u0.w, u1.x, u1.y, u1.z, u1.w};
#pragma unroll
      for (int e = 0; e < 8; ++e) f[e] *= a.scale;
      uint4 hi, lo;
      split_bf16x8(f, hi, lo);
      qh[c] = __builtin_bit_cast(bf16x8_t, hi);
      ql[c] = __builtin_bit_cast(bf16x8_t, lo);
    }
  }
  const int pq = base + j0 + 16 * wave + c16;  // position of this lane's query row
  float m_run = -INFINITY, l_run = 0.f;
  f32x4_t acc_o[ND];
#pragma unroll
  for (int t = 0; t < ND; ++t) acc_o[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  for (int it = 0; 2 * it < n_kt; ++it) {
    const int kt = 2 * it + half;  // this half's tile (past n_kt: none, barriers only)
    const bool live = kt < n_kt;
    __syncthreads();  // the previous tile's reads are done
    if (live) {
      // keys past the context (or on a missing page) stage as zeros: stale entries may hold
      // anything, and a value row enters the products even with probability 0
      if (__any(!kok || !vok[0] || !vok[1])) {
#pragma unroll
        for (int q = 0; q < KF / 4; ++q)
          if (!kok) kr[q] = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
          for (int q = 0; q < VF / 4; ++q)
            if (!vok[u]) vr[u][q] = make_float4(0.f, 0.f, 0.f, 0.f);
      }
#pragma unroll
      for (int q = 0; q < KF / 8; ++q) {
        const float4 u0 = kr[2 * q], u1 = kr[2 * q + 1];
        const float f[8] = {u0.x, u0.y, u0.z, u0.w, u1.x, u1.y, u1.z, u1.w};
        uint4 hi, lo;
        split_bf16x8(f, hi, lo);
        *reinterpret_cast<uint4*>(Ks + (size_t)kk_l * KLD + kd0 + 8 * q) = hi;
        *reinterpret_cast<uint4*>(Ks + (size_t)(KT + kk_l) * KLD + kd0 + 8 * q) = lo;
      }
#pragma unroll
      for (int q = 0; q < VF / 4; ++q) {
        const float a0[4] = {vr[0][q].x, vr[0][q].y, vr[0][q].z, vr[0][q].w};
        const float a1[4] = {vr[1][q].x, vr[1][q].y, vr[1][q].z, vr[1][q].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint32_t hh = pack_bf16x2(a0[e], a1[e]);
          const uint32_t ll = pack_bf16x2(a0[e] - __uint_as_float(hh << 16),
                                          a1[e] - __uint_as_float(hh & 0xffff0000u));
          const int dd = vd0 + 4 * q + e;
          *reinterpret_cast<uint32_t*>(Vt + (size_t)dd * VLD + 2 * vp_l) = hh;
          *reinterpret_cast<uint32_t*>(Vt + (size_t)(DH + dd) * VLD + 2 * vp_l) = ll;
        }
      }
    }
    __syncthreads();
    if (!live) continue;
    if (kt + 2 < n_kt) fetch(kt + 2);

    // scores S^T of the four 16-key sub-tiles; lane: keys 16 st + 4 g + e, query c16
    f32x4_t sc[4];
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      f32x4_t acc = f32x4_t{0.f, 0.f, 0.f, 0.f};
      const bf16_t* kh = Ks + (size_t)(16 * st + c16) * KLD + 8 * g;
      const bf16_t* kl = kh + (size_t)KT * KLD;
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        const bf16x8_t ah = *reinterpret_cast<const bf16x8_t*>(kh + 32 * c);
        const bf16x8_t al = *reinterpret_cast<const bf16x8_t*>(kl + 32 * c);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, qh[c], acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, ql[c], acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, qh[c], acc, 0, 0, 0);
      }
      sc[st] = acc;
    }
    // causal mask (and keys past the context) where the tile reaches the wave's first query
    // position or the end of the context; tile max per query
    if (kt * KT + KT - 1 > base + j0 + 16 * wave || kt * KT + KT > nk) {
#pragma unroll
      for (int st = 0; st < 4; ++st)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int ki = kt * KT + 16 * st + 4 * g + e;
          if (ki > pq || ki >= nk) sc[st][e] = -INFINITY;
        }
    }
    float mt = -INFINITY;
#pragma unroll
    for (int st = 0; st < 4; ++st)
#pragma unroll
      for (int e = 0; e < 4; ++e) mt = fmaxf(mt, sc[st][e]);
    mt = fmaxf(mt, __shfl_xor(mt, 16, SSD_WAVE));
    mt = fmaxf(mt, __shfl_xor(mt, 32, SSD_WAVE));
    const float m_new = fmaxf(m_run, mt);
    const float alpha = m_run == -INFINITY ? 0.f : expf(m_run - m_new);
    float ls = 0.f;
#pragma unroll
    for (int st = 0; st < 4; ++st)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float pv = sc[st][e] == -INFINITY ? 0.f : expf(sc[st][e] - m_new);
        sc[st][e] = pv;
        ls += pv;
      }
    ls += __shfl_xor(ls, 16, SSD_WAVE);
    ls += __shfl_xor(ls, 32, SSD_WAVE);
    l_run = l_run * alpha + ls;
    m_run = m_new;
#pragma unroll
    for (int t = 0; t < ND; ++t) acc_o[t] *= alpha;

    // O^T += V^T . P^T over two 32-key chunks (sub-tiles 2kc, 2kc + 1)
#pragma unroll
    for (int kc = 0; kc < 2; ++kc) {
      float pf[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        pf[e] = sc[2 * kc][e];
        pf[4 + e] = sc[2 * kc + 1][e];
      }
      uint4 phu, plu;
      split_bf16x8(pf, phu, plu);
      const bf16x8_t ph = __builtin_bit_cast(bf16x8_t, phu), pl = __builtin_bit_cast(bf16x8_t, plu);
#pragma unroll
      for (int t = 0; t < ND; ++t) {
        const bf16_t* vh = Vt + (size_t)(16 * t + c16) * VLD + 32 * kc + 4 * g;
        const bf16_t* vl = vh + (size_t)DH * VLD;
        const uint2 h0 = *reinterpret_cast<const uint2*>(vh);
        const uint2 h1 = *reinterpret_cast<const uint2*>(vh + 16);
        const uint2 l0 = *reinterpret_cast<const uint2*>(vl);
        const uint2 l1 = *reinterpret_cast<const uint2*>(vl + 16);
        const bf16x8_t ah = __builtin_bit_cast(bf16x8_t, make_uint4(h0.x, h0.y, h1.x, h1.y));
        const bf16x8_t al = __builtin_bit_cast(bf16x8_t, make_uint4(l0.x, l0.y, l1.x, l1.y));
        acc_o[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, ph, acc_o[t], 0, 0, 0);
        acc_o[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, pl, acc_o[t], 0, 0, 0);
        acc_o[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, ph, acc_o[t], 0, 0, 0);
      }
    }
  }

  // half 1 hands its (max, sum, output) to half 0 through its own stage: lane-major, so that the
  // same (wave, lane) of half 0 reads it back without bank conflicts
  __syncthreads();
  float* xo = reinterpret_cast<float*>(am_s + STAGE) + (size_t)wave * (ND * 4 + 2) * 64;
  if (half == 1) {
#pragma unroll
    for (int t = 0; t < ND; ++t)
#pragma unroll
      for (int e = 0; e < 4; ++e) xo[(4 * t + e) * 64 + lane] = acc_o[t][e];
    xo[ND * 4 * 64 + lane] = m_run;
    xo[(ND * 4 + 1) * 64 + lane] = l_run;
  }
  __syncthreads();
  if (half == 1) return;
  {
    const float m2 = xo[ND * 4 * 64 + lane], l2 = xo[(ND * 4 + 1) * 64 + lane];
    const float m = fmaxf(m_run, m2);
    const float w1 = m_run == -INFINITY ? 0.f : expf(m_run - m);
    const float w2 = m2 == -INFINITY ? 0.f : expf(m2 - m);
    l_run = w1 * l_run + w2 * l2;
#pragma unroll
    for (int t = 0; t < ND; ++t)
#pragma unroll
      for (int e = 0; e < 4; ++e) acc_o[t][e] = w1 * acc_o[t][e] + w2 * xo[(4 * t + e) * 64 + lane];
  }
  // lane: O^T[16 t + 4 g + e][query c16]
  if (16 * wave + c16 < nq) {
    const float inv = l_run > 0.f ? 1.0f / l_run : 0.f;
    float* orow = a.out + (size_t)(b * a.C + j0 + 16 * wave + c16) * HD + h * DH;
#pragma unroll
    for (int t = 0; t < ND; ++t)
      *reinterpret_cast<float4*>(orow + 16 * t + 4 * g) =
          make_float4(acc_o[t][0] * inv, acc_o[t][1] * inv, acc_o[t][2] * inv, acc_o[t][3] * inv);
  }
}

// LDS limit of attn_mfma_kernel (one block a compute unit: two 68 KB stages at dh 128 and the
// page-table entries of up to 5120 pages)
constexpr int ATTN_MFMA_LDS = 156 * 1024;

// LDS of attn_mfma_kernel: the K and V^T planes, then one page-table entry per page of max_seq.
template <int DH>
size_t attn_mfma_shm(const AttnArgs& a) {
  const size_t stage = ((size_t)2 * 64 * (DH + 8) + (size_t)2 * DH * (64 + 4)) * sizeof(bf16_t);
  return 2 * stage + (size_t)((a.max_seq + a.kv.page_size - 1) / a.kv.page_size) * sizeof(int);
}

// The MFMA prefill attention applies: self-attention of more than 16 rows a sequence over a
// float32 cache whose pages hold 2..64 keys dividing 64, no position bias, no output planes.
bool attn_mfma_ok(const AttnArgs& a) {
  if (a.cross || a.C <= 16 || a.kvdtype != 0 || a.bias || a.out_planes || a.kv.page_size < 2 ||
      64 % a.kv.page_size || (a.dh != 64 && a.dh != 128))
    return false;
  const size_t shm = a.dh == 64 ? attn_mfma_shm<64>(a) : attn_mfma_shm<128>(a);
  return shm <= (size_t)ATTN_MFMA_LDS;
}

template <int DH>
hipError_t launch_attn_mfma(const AttnArgs& a, hipStream_t s) {
  const size_t shm = attn_mfma_shm<DH>(a);
  // the attribute is raised once to the largest size any launch may take (ATTN_MFMA_LDS)
  static bool attr = false;
  if (!attr) {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&attn_mfma_kernel<DH>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, ATTN_MFMA_LDS);
    attr = true;
  }
  const int n_qt = (a.C + 63) / 64;
  hipLaunchKernelGGL((attn_mfma_kernel<DH>), dim3(n_qt, a.H, a.B), dim3(512), shm, s, a, n_qt);
  return hipGetLastError();
}

// One key split of a verify chunk's causal self-attention on MFMA (float32 cache, no position
// bias; a chunk of at most 16 rows over a long context): one block of four waves per (head,
// sequence, key split).  The split's keys are staged 128 at a time in LDS as bf16 hi / lo planes
// (K by key row, V transposed); wave w takes keys 32w..32w+31 of each tile for all the chunk's
// rows, with the scores S^T = K . Q^T and the output O^T += V^T . P^T of attn_mfma_kernel and a
// running max and sum per query lane.  The four waves' triples are merged through LDS into the
// split's partial (unnormalised output, max, sum), which attn_combine_kernel merges over the
// splits as it does for attn_kernel.
template <int DH>
__global__ __launch_bounds__(256) void attn_mfma_chunk_kernel(const AttnArgs a, const int ks) {
  constexpr int KT = 128;       // keys per tile
  constexpr int KLD = DH + 8;   // bf16 per key row of the K planes
  constexpr int VLD = KT + 4;   // bf16 per dimension row of the V^T planes (66 dwords: the
                                // transposed stores of a wave hit 64 distinct banks)
  constexpr int NC = DH / 32, ND = DH / 16;
  constexpr int KF = DH / 2;    // K floats a thread stages (2 threads per key)
  constexpr int VF = DH / 4;    // V floats per key a thread stages (4 threads per key pair)
  extern __shared__ __attribute__((aligned(16))) bf16_t ac_s[];
  bf16_t* Ks = ac_s;                   // [2][KT][KLD]
  bf16_t* Vt = ac_s + 2 * KT * KLD;    // [2][DH][VLD]
  int* pg = reinterpret_cast<int*>(Vt + 2 * DH * VLD);

  const int h = blockIdx.x, b = blockIdx.y, split = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, c16 = lane & 15;
  const int C = a.C, HD = a.H * DH, ps = a.kv.page_size;
  const int base = a.kv.seq_len[b] + a.kv.pos_off;
  int nk_all = base + C;
  if (nk_all > a.max_seq) {
    if (tid == 0 && split == 0) atomicOr(a.status, SSD_DEV_CAPACITY);
    nk_all = a.max_seq;
  }
  const int kfix = (a.max_seq + ks - 1) / ks;
  const int k0 = split * kfix, k_end = min(nk_all, k0 + kfix);
  const int nks = k_end > k0 ? k_end - k0 : 0;
  const int p0 = k0 / ps;
  const int n_pg = nks > 0 ? (k_end - 1) / ps - p0 + 1 : 0;
  for (int i = tid; i < n_pg; i += 256)
    pg[i] = p0 + i < a.kv.max_pages ? a.kv.page_table[(size_t)b * a.kv.max_pages + p0 + i] : -1;

  // the chunk's rows as the B operand (hi / lo), pre-scaled; rows past C repeat the last
  const int jq = min(c16, C - 1);
  bf16x8_t qh[NC], ql[NC];
  {
    const float* qrow = a.q + (size_t)(b * C + jq) * HD + h * DH;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const float4 u0 = reinterpret_cast<const float4*>(qrow + 32 * c + 8 * g)[0];
      const float4 u1 = reinterpret_cast<const float4*>(qrow + 32 * c + 8 * g)[1];
      float f[8] = {u0.x, u0.y, u0.z, u0.w, u1.x, u1.y, u1.z, u1.w};
#pragma unroll
      for (int e = 0; e < 8; ++e) f[e] *= a.scale;
      uint4 hi, lo;
      split_bf16x8(f, hi, lo);
      qh[c] = __builtin_bit_cast(bf16x8_t, hi);
      ql[c] = __builtin_bit_cast(bf16x8_t, lo);
    }
  }
  const int pq = base + jq;
  float m_run = -INFINITY, l_run = 0.f;
  f32x4_t acc_o[ND];
#pragma unroll
  for (int t = 0; t < ND; ++t) acc_o[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  const float* Kp = reinterpret_cast<const float*>(a.kv.k);
  const float* Vp = reinterpret_cast<const float*>(a.kv.v);
  const int kk_l = tid >> 1, kd0 = (tid & 1) * KF;   // K staging: key, first float
  const int vp_l = tid & 63, vd0 = (tid >> 6) * VF;  // V staging: key pair, first float
  __syncthreads();  // page entries

  for (int t0 = 0; t0 < nks; t0 += KT) {
    if (t0 > 0) __syncthreads();  // the previous tile's reads are done
    {
      // key ki = k0 + t0 + key of the tile: its page entry pg[ki / ps - p0]; keys past the split
      // (or on a missing page) stage as zeros
      int ki = k0 + t0 + kk_l;
      bool ok = ki < k_end;
      int pe = pg[min(ki, k_end - 1) / ps - p0];
      ok = ok && pe >= 0 && pe < a.kv.n_pages;
      const float* src = Kp + (((size_t)(ok ? pe : 0) * a.H + h) * ps + (ok ? ki % ps : 0)) * DH + kd0;
#pragma unroll
      for (int q = 0; q < KF / 8; ++q) {
        const float4 u0 = ok ? reinterpret_cast<const float4*>(src)[2 * q] : make_float4(0.f, 0.f, 0.f, 0.f);
        const float4 u1 = ok ? reinterpret_cast<const float4*>(src)[2 * q + 1] : make_float4(0.f, 0.f, 0.f, 0.f);
        const float f[8] = {u0.x, u0.y, u0.z, u0.w, u1.x, u1.y, u1.z, u1.w};
        uint4 hi, lo;
        split_bf16x8(f, hi, lo);
        *reinterpret_cast<uint4*>(Ks + (size_t)kk_l * KLD + kd0 + 8 * q) = hi;
        *reinterpret_cast<uint4*>(Ks + (size_t)(KT + kk_l) * KLD + kd0 + 8 * q) = lo;
      }
      float4 vr[2][VF / 4];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        ki = k0 + t0 + 2 * vp_l + u;
        ok = ki < k_end;
        pe = pg[min(ki, k_end - 1) / ps - p0];
        ok = ok && pe >= 0 && pe < a.kv.n_pages;
        const float* vs = Vp + (((size_t)(ok ? pe : 0) * a.H + h) * ps + (ok ? ki % ps : 0)) * DH + vd0;
#pragma unroll
        for (int q = 0; q < VF / 4; ++q)
          vr[u][q] = ok ? reinterpret_cast<const float4*>(vs)[q] : make_float4(0.f, 0.f, 0.f, 0.f);
      }
#pragma unroll
      for (int q = 0; q < VF / 4; ++q) {
        const float a0[4] = {vr[0][q].x, vr[0][q].y, vr[0][q].z, vr[0][q].w};
        const float a1[4] = {vr[1][q].x, vr[1][q].y, vr[1][q].z, vr[1][q].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint32_t hh = pack_bf16x2(a0[e], a1[e]);
          const uint32_t ll = pack_bf16x2(a0[e] - __uint_as_float(hh << 16),
                                          a1[e] - __uint_as_float(hh & 0xffff0000u));
          const int dd = vd0 + 4 * q + e;
          *reinterpret_cast<uint32_t*>(Vt + (size_t)dd * VLD + 2 * vp_l) = hh;
          *reinterpret_cast<uint32_t*>(Vt + (size_t)(DH + dd) * VLD + 2 * vp_l) = ll;
        }
      }
    }
    __syncthreads();

    // this wave's two 16-key sub-tiles (keys 32 wave + 16 s + 4 g + e of the tile)
    f32x4_t sc[2];
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      f32x4_t acc = f32x4_t{0.f, 0.f, 0.f, 0.f};
      const bf16_t* kh = Ks + (size_t)(32 * wave + 16 * s2 + c16) * KLD + 8 * g;
      const bf16_t* kl = kh + (size_t)KT * KLD;
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        const bf16x8_t ah = *reinterpret_cast<const bf16x8_t*>(kh + 32 * c);
        const bf16x8_t al = *reinterpret_cast<const bf16x8_t*>(kl + 32 * c);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, qh[c], acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, ql[c], acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, qh[c], acc, 0, 0, 0);
      }
      sc[s2] = acc;
    }
    float mt = -INFINITY;
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int ki = k0 + t0 + 32 * wave + 16 * s2 + 4 * g + e;
        if (ki >= k_end || ki > pq) sc[s2][e] = -INFINITY;
        mt = fmaxf(mt, sc[s2][e]);
      }
    mt = fmaxf(mt, __shfl_xor(mt, 16, SSD_WAVE));
    mt = fmaxf(mt, __shfl_xor(mt, 32, SSD_WAVE));
    const float m_new = fmaxf(m_run, mt);
    const float alpha = m_run == -INFINITY ? 0.f : expf(m_run - m_new);
    float ls = 0.f, pf[8];
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float pv = sc[s2][e] == -INFINITY ? 0.f : expf(sc[s2][e] - m_new);
        pf[4 * s2 + e] = pv;
        ls += pv;
      }
    ls += __shfl_xor(ls, 16, SSD_WAVE);
    ls += __shfl_xor(ls, 32, SSD_WAVE);
    l_run = l_run * alpha + ls;
    m_run = m_new;
    uint4 phu, plu;
    split_bf16x8(pf, phu, plu);
    const bf16x8_t ph = __builtin_bit_cast(bf16x8_t, phu), pl = __builtin_bit_cast(bf16x8_t, plu);
#pragma unroll
    for (int t = 0; t < ND; ++t) {
      acc_o[t] *= alpha;
      const bf16_t* vh = Vt + (size_t)(16 * t + c16) * VLD + 32 * wave + 4 * g;
      const bf16_t* vl = vh + (size_t)DH * VLD;
      const uint2 h0 = *reinterpret_cast<const uint2*>(vh);
      const uint2 h1 = *reinterpret_cast<const uint2*>(vh + 16);
      const uint2 l0 = *reinterpret_cast<const uint2*>(vl);
      const uint2 l1 = *reinterpret_cast<const uint2*>(vl + 16);
      const bf16x8_t ah = __builtin_bit_cast(bf16x8_t, make_uint4(h0.x, h0.y, h1.x, h1.y));
      const bf16x8_t al = __builtin_bit_cast(bf16x8_t, make_uint4(l0.x, l0.y, l1.x, l1.y));
      acc_o[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, ph, acc_o[t], 0, 0, 0);
      acc_o[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, pl, acc_o[t], 0, 0, 0);
      acc_o[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, ph, acc_o[t], 0, 0, 0);
    }
  }

  // merge the four waves' (max, sum, output) through LDS (lane-major), then the split's partial
  __syncthreads();
  float* xo = reinterpret_cast<float*>(ac_s);
  float* mine = xo + (size_t)wave * (ND * 4 + 2) * 64;
#pragma unroll
  for (int t = 0; t < ND; ++t)
#pragma unroll
    for (int e = 0; e < 4; ++e) mine[(4 * t + e) * 64 + lane] = acc_o[t][e];
  mine[ND * 4 * 64 + lane] = m_run;
  mine[(ND * 4 + 1) * 64 + lane] = l_run;
  __syncthreads();
  if (wave != 0 || c16 >= C) return;
  float mw[4], M = -INFINITY;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    mw[w] = xo[(size_t)w * (ND * 4 + 2) * 64 + ND * 4 * 64 + lane];
    M = fmaxf(M, mw[w]);
  }
  float fw[4], L = 0.f;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    fw[w] = mw[w] == -INFINITY ? 0.f : expf(mw[w] - M);
    L = fmaf(fw[w], xo[(size_t)w * (ND * 4 + 2) * 64 + (ND * 4 + 1) * 64 + lane], L);
  }
  float* pp = a.part + (((size_t)(b * C + c16) * a.H + h) * ks + split) * (DH + 2);
#pragma unroll
  for (int t = 0; t < ND; ++t) {
    float o4[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float v = 0.f;
#pragma unroll
      for (int w = 0; w < 4; ++w) v = fmaf(fw[w], xo[(size_t)w * (ND * 4 + 2) * 64 + (4 * t + e) * 64 + lane], v);
      o4[e] = v;
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) pp[16 * t + 4 * g + e] = o4[e];
  }
  if (g == 0) {
    pp[DH] = M;
    pp[DH + 1] = L;
  }
}

// LDS of attn_mfma_chunk_kernel: the K and V^T planes of a 128-key tile, then the page entries of
// one split's keys.
template <int DH>
size_t attn_chunk_shm(const AttnArgs& a, int ks) {
  const size_t planes = ((size_t)2 * 128 * (DH + 8) + (size_t)2 * DH * (128 + 4)) * sizeof(bf16_t);
  const int kfix = (a.max_seq + ks - 1) / ks;
  return planes + (size_t)(kfix / a.kv.page_size + 2) * sizeof(int);
}

// The MFMA chunk attention applies: self-attention of 2..16 rows a sequence over a long float32
// cache split into ks > 1 key ranges (partials merged by attn_combine_kernel), even pages, no
// position bias.
bool attn_chunk_ok(const AttnArgs& a, int ks) {
  if (a.cross || a.C < 2 || a.C > 16 || ks < 2 || a.kvdtype != 0 || a.bias || !a.part ||
      a.kv.page_size < 2 || (a.dh != 64 && a.dh != 128))
    return false;
  const size_t shm = a.dh == 64 ? attn_chunk_shm<64>(a, ks) : attn_chunk_shm<128>(a, ks);
  return shm <= (size_t)156 * 1024;
}

template <int DH>
void launch_attn_chunk(const AttnArgs& a, int ks, hipStream_t s) {
  static bool attr = false;
  if (!attr) {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&attn_mfma_chunk_kernel<DH>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, 156 * 1024);
    attr = true;
  }
  hipLaunchKernelGGL((attn_mfma_chunk_kernel<DH>), dim3(a.H, a.B, ks), dim3(256),
                     attn_chunk_shm<DH>(a, ks), s, a, ks);
}

// Key splits of a launch with `groups` query blocks per sequence: long self-attention contexts
// (capacity of 256 keys and more, up to 16 query rows) are split so that about 512 blocks share
// the keys, at least 128 keys a split.
int attn_splits(const AttnArgs& a, int groups) {
  if (a.cross || a.C > 16 || !a.part || a.B * a.C > a.part_rows || a.max_seq < 256) return 1;
  const int blocks = a.H * a.B * groups;
  const int want = (512 + blocks - 1) / blocks;
  const int by_len = (a.max_seq + 127) / 128;
  int ks = want < by_len ? want : by_len;
  if (ks > ATTN_SPLITS_MAX) ks = ATTN_SPLITS_MAX;
  return ks < 1 ? 1 : ks;
}

template <typename KT, int DH>
hipError_t launch_attn_dh(const AttnArgs& a, hipStream_t s) {
  const int nk_max = a.cross ? a.n_keys : a.max_seq;
  const bool long_ctx = !a.cross && a.max_seq >= 256;
  const bool rs = attn_pool_bytes<KT, DH>(a) <= ATTN_RS_MAX;
  int ks = 1;
  if (a.C == 1 || (a.C <= 16 && !long_ctx)) {
    // decode steps and short-context verify chunks: one block per (head, sequence, query row
    // [, key split]); the rows of a chunk re-read the same few keys from L2, and more blocks keep
    // the chip busy
    ks = attn_splits(a, a.C);
    const int s_stride = (((nk_max + ks - 1) / ks) + 63) & ~63;
    dim3 grid(a.H, a.B, a.C * ks);
    const size_t shm = (size_t)s_stride * sizeof(float);
    if (rs)
      hipLaunchKernelGGL((attn_kernel<KT, DH, 1, true>), grid, dim3(256), shm, s, a, s_stride, ks);
    else
      hipLaunchKernelGGL((attn_kernel<KT, DH, 1, false>), grid, dim3(256), shm, s, a, s_stride, ks);
  } else {
    // prefill blocks and long-context verify chunks: up to QB rows of a sequence share each key
    // load (and long contexts split their keys)
    const int groups = (a.C + QB - 1) / QB;
    ks = attn_splits(a, groups);
    const int s_stride = (((nk_max + ks - 1) / ks) + 63) & ~63;
    dim3 grid(a.H, a.B, groups * ks);
    const size_t shm = (size_t)QB * s_stride * sizeof(float);
    if (sizeof(KT) == 4 && attn_chunk_ok(a, ks))
      launch_attn_chunk<DH>(a, ks, s);
    else if (rs)
      hipLaunchKernelGGL((attn_kernel<KT, DH, QB, true>), grid, dim3(256), shm, s, a, s_stride, ks);
    else
      hipLaunchKernelGGL((attn_kernel<KT, DH, QB, false>), grid, dim3(256), shm, s, a, s_stride, ks);
  }
  if (ks > 1) {
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((attn_combine_kernel<DH>), dim3(a.H, a.B * a.C), dim3(DH), 0, s, a, ks);
  }
  return hipGetLastError();
}

template <typename KT>
hipError_t launch_attn_t(const AttnArgs& a, hipStream_t s) {
  if (attn_mfma_ok(a)) return a.dh == 64 ? launch_attn_mfma<64>(a, s) : launch_attn_mfma<128>(a, s);
  return a.dh == 64 ? launch_attn_dh<KT, 64>(a, s) : launch_attn_dh<KT, 128>(a, s);
}

// Folded cross-attention, query side: fq[h*NV + j][k] = sum_e K[h][j][e] * Wq[h*dh + e][k].
// Block (column tile of 512, head h): lane l of every wave owns columns 8l .. 8l + 7 of the tile
// (one 16-byte load of Wq per e) and wave w the keys j = w, w + 4, ... (the four waves read the
// same weights, from L2 after the first); the head's keys sit in LDS.
template <typename KT, typename WT, int NV>
__global__ __launch_bounds__(256) void fold_q_kernel(const KT* __restrict__ xk,
                                                     const WT* __restrict__ wq, float* __restrict__ fq,
                                                     int dh, int d) {
  constexpr int JW = (NV + 3) / 4;  // keys per wave
  __shared__ __attribute__((aligned(16))) float ks[NV][128 + 4];
  const int h = blockIdx.y, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int k = blockIdx.x * 512 + lane * 8;
  for (int i = threadIdx.x; i < NV * dh; i += 256) {
    const int j = i / dh, e = i - j * dh;
    ks[j][e] = load_elem(xk + ((size_t)h * NV + j) * dh + e);
  }
  __syncthreads();
  if (k >= d) return;  // d is a multiple of 8
  float acc[JW][8];
#pragma unroll
  for (int t = 0; t < JW; ++t)
#pragma unroll
    for (int c = 0; c < 8; ++c) acc[t][c] = 0.f;
  // EB rows of Wq requested at once (dh is a multiple of 16), then their products
  constexpr int EB = NV >= 64 ? 8 : 16;
  for (int e0 = 0; e0 < dh; e0 += EB) {
    Vec8<WT> v8[EB];
#pragma unroll
    for (int u = 0; u < EB; ++u) v8[u].load(wq + ((size_t)h * dh + e0 + u) * d + k);
#pragma unroll
    for (int u = 0; u < EB; ++u) {
      float w[8];
      v8[u].to_f32(w);
#pragma unroll
      for (int t = 0; t < JW; ++t) {
        const int j = wave + 4 * t;
        const float kv = j < NV ? ks[j][e0 + u] : 0.f;
#pragma unroll
        for (int c = 0; c < 8; ++c) acc[t][c] = fmaf(kv, w[c], acc[t][c]);
      }
    }
  }
#pragma unroll
  for (int t = 0; t < JW; ++t) {
    const int j = wave + 4 * t;
    if (j >= NV) continue;
    float* dst = fq + ((size_t)h * NV + j) * d + k;
    *reinterpret_cast<float4*>(dst) = make_float4(acc[t][0], acc[t][1], acc[t][2], acc[t][3]);
    *reinterpret_cast<float4*>(dst + 4) = make_float4(acc[t][4], acc[t][5], acc[t][6], acc[t][7]);
  }
}

// Folded cross-attention, output side: fo[n][h*NV + j] = sum_e Wo[n][h*dh + e] * V[h][j][e].
// Block (row tile, head h): thread t owns output row n and reads its dh weights of head h (a
// contiguous run, eight elements per load); the head's values sit in LDS, read four e at a time.
template <typename KT, typename WT, int NV>
__global__ __launch_bounds__(256) void fold_o_kernel(const KT* __restrict__ xv,
                                                     const WT* __restrict__ wo, float* __restrict__ fo,
                                                     int H, int dh, int d) {
  __shared__ __attribute__((aligned(16))) float vs[NV][128 + 4];
  const int h = blockIdx.y, n = blockIdx.x * 256 + threadIdx.x;
  for (int i = threadIdx.x; i < NV * dh; i += 256) {
    const int j = i / dh, e = i - j * dh;
    vs[j][e] = load_elem(xv + ((size_t)h * NV + j) * dh + e);
  }
  __syncthreads();
  if (n >= d) return;
  const int HD = H * dh;
  const WT* wr = wo + (size_t)n * HD + (size_t)h * dh;
  float acc[NV];
#pragma unroll
  for (int j = 0; j < NV; ++j) acc[j] = 0.f;
  // OB pieces of eight of the row's dh weights requested at once (dh is 64 or 128), then their
  // products
  constexpr int OB = NV >= 64 ? 4 : 8;
  for (int p0 = 0; p0 * 8 < dh; p0 += OB) {
  Vec8<WT> v8[OB];
#pragma unroll
  for (int u = 0; u < OB; ++u)
    if ((p0 + u) * 8 < dh) v8[u].load(wr + (p0 + u) * 8);
#pragma unroll
  for (int u = 0; u < OB; ++u) {
    if ((p0 + u) * 8 >= dh) break;
    const int e0 = (p0 + u) * 8;
    float w[8];
    v8[u].to_f32(w);
#pragma unroll
    for (int j = 0; j < NV; ++j) {
      const float4 a0 = *reinterpret_cast<const float4*>(&vs[j][e0]);
      const float4 a1 = *reinterpret_cast<const float4*>(&vs[j][e0 + 4]);
      float t = acc[j];
      t = fmaf(a0.x, w[0], t); t = fmaf(a0.y, w[1], t); t = fmaf(a0.z, w[2], t); t = fmaf(a0.w, w[3], t);
      t = fmaf(a1.x, w[4], t); t = fmaf(a1.y, w[5], t); t = fmaf(a1.z, w[6], t); t = fmaf(a1.w, w[7], t);
      acc[j] = t;
    }
  }
  }
  float* dst = fo + (size_t)n * H * NV + (size_t)h * NV;
#pragma unroll
  for (int j = 0; j < NV; ++j) dst[j] = acc[j];
}

template <typename KT, typename WT, int NV>
hipError_t launch_fold_t(const void* xk, const void* xv, const void* wq, const void* wo, int H,
                         int dh, int d, float* fq, float* fo, hipStream_t s) {
  const dim3 grid((d + 255) / 256, H);
  hipLaunchKernelGGL((fold_q_kernel<KT, WT, NV>), dim3((d + 511) / 512, H), dim3(256), 0, s,
                     reinterpret_cast<const KT*>(xk), reinterpret_cast<const WT*>(wq), fq, dh, d);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((fold_o_kernel<KT, WT, NV>), grid, dim3(256), 0, s,
                     reinterpret_cast<const KT*>(xv), reinterpret_cast<const WT*>(wo), fo, H, dh, d);
  return hipGetLastError();
}

template <int NV>
hipError_t launch_fold_nv(const void* xk, const void* xv, int kvdtype, const void* wq,
                          const void* wo, int wdtype, int H, int dh, int d, float* fq, float* fo,
                          hipStream_t s) {
  if (kvdtype == 1)
    return wdtype == 1 ? launch_fold_t<bf16_t, bf16_t, NV>(xk, xv, wq, wo, H, dh, d, fq, fo, s)
                       : launch_fold_t<bf16_t, float, NV>(xk, xv, wq, wo, H, dh, d, fq, fo, s);
  return wdtype == 1 ? launch_fold_t<float, bf16_t, NV>(xk, xv, wq, wo, H, dh, d, fq, fo, s)
                     : launch_fold_t<float, float, NV>(xk, xv, wq, wo, H, dh, d, fq, fo, s);
}

}  // namespace

// fg[j][n] = fold_q[j][n] g[n] for n < d; fg[j][d + c] = sum_n fold_q[j][n] g[n] wo[n][c].
// A 64 x 64 tile of the product per block on v_mfma_f32_16x16x32_bf16: each wave owns 32 x 32
// (2 x 2 MFMA tiles).  Per K step of 64 the scaled fold_q rows are split into bf16 hi / lo planes
// in LDS (two MFMAs, about 16 mantissa bits) and the W_o rows are stored transposed, so that both
// operand fragments are 16-byte LDS reads; the next step's global loads are issued before the
// current step's MFMAs.  Rows, columns and K past the matrix read as zeros.
template <typename WT>
struct FgRegs {
  float a[16];   // fold_q[row][k .. k + 16) * g[k ..]
  float b[16];   // wo[k row][c .. c + 16)
};

template <typename WT>
__device__ __forceinline__ void fg_load(FgRegs<WT>& r, const float* __restrict__ fq,
                                        const float* __restrict__ g, const WT* __restrict__ wo,
                                        int HN, int d, int HD, int jrow, int kcol, int krow,
                                        int ccol) {
  if (jrow < HN && kcol + 16 <= d) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const float4 v = *reinterpret_cast<const float4*>(fq + (size_t)jrow * d + kcol + 4 * u);
      const float4 w = *reinterpret_cast<const float4*>(g + kcol + 4 * u);
      r.a[4 * u] = v.x * w.x; r.a[4 * u + 1] = v.y * w.y;
      r.a[4 * u + 2] = v.z * w.z; r.a[4 * u + 3] = v.w * w.w;
    }
  } else {
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int k = kcol + e;
      r.a[e] = (jrow < HN && k < d) ? fq[(size_t)jrow * d + k] * g[k] : 0.f;
    }
  }
  if (krow < d && ccol + 16 <= HD) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      Vec8<WT> v;
      v.load(wo + (size_t)krow * HD + ccol + 8 * u);
      v.to_f32(r.b + 8 * u);
    }
  } else {
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int c = ccol + e;
      r.b[e] = (krow < d && c < HD) ? load_elem(wo + (size_t)krow * HD + c) : 0.f;
    }
  }
}

template <typename WT>
__global__ __launch_bounds__(256) void fold_fg_kernel(const float* __restrict__ fq,
                                                      const float* __restrict__ g,
                                                      const WT* __restrict__ wo, int HN, int d,
                                                      int HD, float* __restrict__ fg) {
  constexpr int KS = 64, LDK = KS + 8;  // K per step; bf16 per LDS row (with padding)
  __shared__ __attribute__((aligned(16))) bf16_t Ah[64 * LDK], Al[64 * LDK], Bt[64 * LDK];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int j0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
  const int wr = (wave >> 1) * 32, wc = (wave & 1) * 32;
  const size_t ldg = (size_t)d + HD;
  f32x4_t acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) acc[a][b] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  const int ar = tid >> 2, ak = (tid & 3) * 16;  // A: row, first K element of this thread
  const int bk = tid >> 2, bc = (tid & 3) * 16;  // B: K row, first column of this thread
  FgRegs<WT> r;
  fg_load(r, fq, g, wo, HN, d, HD, j0 + ar, ak, bk, c0 + bc);
  for (int n0 = 0; n0 < d; n0 += KS) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      uint4 hi, lo;
      split_bf16x8(r.a + 8 * h, hi, lo);
      *reinterpret_cast<uint4*>(Ah + ar * LDK + ak + 8 * h) = hi;
      *reinterpret_cast<uint4*>(Al + ar * LDK + ak + 8 * h) = lo;
    }
#pragma unroll
    for (int e = 0; e < 16; ++e) Bt[(bc + e) * LDK + bk] = (bf16_t)f32_to_bf16(r.b[e]);
    __syncthreads();
    if (n0 + KS < d) fg_load(r, fq, g, wo, HN, d, HD, j0 + ar, n0 + KS + ak, n0 + KS + bk, c0 + bc);
#pragma unroll
    for (int kk = 0; kk < KS; kk += 32) {
      const int kq = kk + 8 * (lane >> 4);
#pragma unroll
      for (int a = 0; a < 2; ++a) {
        const int row = wr + 16 * a + (lane & 15);
        const bf16x8_t ah = *reinterpret_cast<const bf16x8_t*>(Ah + row * LDK + kq);
        const bf16x8_t al = *reinterpret_cast<const bf16x8_t*>(Al + row * LDK + kq);
#pragma unroll
        for (int b = 0; b < 2; ++b) {
          const int col = wc + 16 * b + (lane & 15);
          const bf16x8_t bv = *reinterpret_cast<const bf16x8_t*>(Bt + col * LDK + kq);
          acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bv, acc[a][b], 0, 0, 0);
          acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, bv, acc[a][b], 0, 0, 0);
        }
      }
    }
    __syncthreads();
  }
  // D[row][col]: lane holds rows 4 (lane / 16) + e, column lane % 16 of each tile
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int j = j0 + wr + 16 * a + 4 * (lane >> 4) + e, c = c0 + wc + 16 * b + (lane & 15);
        if (j < HN && c < HD) fg[(size_t)j * ldg + d + c] = acc[a][b][e];
      }
  // the scaled F part: row j0 + jr goes to the column block jr % gridDim.x (d % 4 == 0)
  for (int jr = blockIdx.x; jr < 64; jr += gridDim.x) {
    const int j = j0 + jr;
    if (j >= HN) break;
    for (int n = tid * 4; n < d; n += 1024) {
      const float4 v = *reinterpret_cast<const float4*>(fq + (size_t)j * d + n);
      const float4 w = *reinterpret_cast<const float4*>(g + n);
      float* o = fg + (size_t)j * ldg + n;
      o[0] = v.x * w.x; o[1] = v.y * w.y; o[2] = v.z * w.z; o[3] = v.w * w.w;
    }
  }
}

bool cross_fold_ok(int nv, int dh) {
  return (nv == 8 || nv == 16 || nv == 32 || nv == 64) && dh <= 128;
}

hipError_t launch_fold_fg(const float* fold_q, const float* gain, const void* wo, int wdtype,
                          int HN, int d, int HD, float* fg, hipStream_t s) {
  if (HN < 1 || d < 1 || HD < 1) return hipErrorInvalidValue;
  dim3 grid((HD + 63) / 64, (HN + 63) / 64);
  if (wdtype == 1)
    hipLaunchKernelGGL(fold_fg_kernel<bf16_t>, grid, dim3(256), 0, s, fold_q, gain,
                       reinterpret_cast<const bf16_t*>(wo), HN, d, HD, fg);
  else
    hipLaunchKernelGGL(fold_fg_kernel<float>, grid, dim3(256), 0, s, fold_q, gain,
                       reinterpret_cast<const float*>(wo), HN, d, HD, fg);
  return hipGetLastError();
}

hipError_t launch_cross_fold(const void* xk, const void* xv, int kvdtype, const void* wq,
                             const void* wo, int wdtype, int H, int nv, int dh, int d, float* fq,
                             float* fo, hipStream_t s) {
  if (!cross_fold_ok(nv, dh) || H < 1 || d < 1 || d % 8) return hipErrorInvalidValue;
  switch (nv) {
    case 8: return launch_fold_nv<8>(xk, xv, kvdtype, wq, wo, wdtype, H, dh, d, fq, fo, s);
    case 16: return launch_fold_nv<16>(xk, xv, kvdtype, wq, wo, wdtype, H, dh, d, fq, fo, s);
    case 32: return launch_fold_nv<32>(xk, xv, kvdtype, wq, wo, wdtype, H, dh, d, fq, fo, s);
    default: return launch_fold_nv<64>(xk, xv, kvdtype, wq, wo, wdtype, H, dh, d, fq, fo, s);
  }
}

hipError_t launch_attention(const AttnArgs& a, hipStream_t s) {
  if (a.B <= 0 || a.C <= 0) return hipSuccess;
  return a.kvdtype == 1 ? launch_attn_t<bf16_t>(a, s) : launch_attn_t<float>(a, s);
}

}  // namespace ssd
