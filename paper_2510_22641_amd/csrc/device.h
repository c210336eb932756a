// Device helpers shared by the gfx950 kernels: bf16 conversion, wave reductions, activations.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#define SSD_WAVE 64

typedef uint16_t bf16_t;  // bfloat16 storage (same typedef as kernels.h)

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_to_f32(uint32_t h) { return __uint_as_float(h << 16); }

// float -> bfloat16, round to nearest even (NaN kept quiet): gfx950's v_cvt_pk_bf16_f32
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
  return __builtin_bit_cast(uint16_t, (__bf16)f);
}

// Two floats -> two bfloat16 (a in the low half), one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  typedef __bf16 bf16x2_v __attribute__((ext_vector_type(2)));
  const bf16x2_v v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}

// Unpack a 16-byte vector of 8 bf16 into floats.
__device__ __forceinline__ void unpack_bf16x8(const uint4& r, float* f) {
  f[0] = __uint_as_float(r.x << 16); f[1] = __uint_as_float(r.x & 0xffff0000u);
  f[2] = __uint_as_float(r.y << 16); f[3] = __uint_as_float(r.y & 0xffff0000u);
  f[4] = __uint_as_float(r.z << 16); f[5] = __uint_as_float(r.z & 0xffff0000u);
  f[6] = __uint_as_float(r.w << 16); f[7] = __uint_as_float(r.w & 0xffff0000u);
}

// Split eight floats into bf16 planes hi = bf16(f), lo = bf16(f - hi): hi + lo carries about 16
// mantissa bits, so two bf16 MFMAs over (hi, lo) act on near-fp32 activations.
__device__ __forceinline__ void split_bf16x8(const float* f, uint4& hi, uint4& lo) {
  uint32_t h[4], l[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    h[e] = pack_bf16x2(f[2 * e], f[2 * e + 1]);
    l[e] = pack_bf16x2(f[2 * e] - __uint_as_float(h[e] << 16),
                       f[2 * e + 1] - __uint_as_float(h[e] & 0xffff0000u));
  }
  hi = make_uint4(h[0], h[1], h[2], h[3]);
  lo = make_uint4(l[0], l[1], l[2], l[3]);
}

// split_bf16x8 on values: hi / lo bf16 of the eight floats (a0.x .. a1.w).
__device__ __forceinline__ void split_bf16x8_v(const float4& a0, const float4& a1, uint4& hi, uint4& lo) {
  const uint32_t h0 = pack_bf16x2(a0.x, a0.y), h1 = pack_bf16x2(a0.z, a0.w);
  const uint32_t h2 = pack_bf16x2(a1.x, a1.y), h3 = pack_bf16x2(a1.z, a1.w);
  hi = make_uint4(h0, h1, h2, h3);
  lo = make_uint4(pack_bf16x2(a0.x - __uint_as_float(h0 << 16), a0.y - __uint_as_float(h0 & 0xffff0000u)),
                  pack_bf16x2(a0.z - __uint_as_float(h1 << 16), a0.w - __uint_as_float(h1 & 0xffff0000u)),
                  pack_bf16x2(a1.x - __uint_as_float(h2 << 16), a1.y - __uint_as_float(h2 & 0xffff0000u)),
                  pack_bf16x2(a1.z - __uint_as_float(h3 << 16), a1.w - __uint_as_float(h3 & 0xffff0000u)));
}

// Eight consecutive elements of a weight (or KV) row, as raw registers until converted.
template <typename T> struct Vec8;
template <> struct Vec8<bf16_t> {
  uint4 r;
  __device__ __forceinline__ void load(const bf16_t* p) { r = *reinterpret_cast<const uint4*>(p); }
  __device__ __forceinline__ void zero() { r = make_uint4(0, 0, 0, 0); }
  __device__ __forceinline__ void to_f32(float* f) const { unpack_bf16x8(r, f); }
};
template <> struct Vec8<float> {
  float4 a, b;
  __device__ __forceinline__ void load(const float* p) {
    a = reinterpret_cast<const float4*>(p)[0];
    b = reinterpret_cast<const float4*>(p)[1];
  }
  __device__ __forceinline__ void zero() { a = b = make_float4(0.f, 0.f, 0.f, 0.f); }
  __device__ __forceinline__ void to_f32(float* f) const {
    f[0] = a.x; f[1] = a.y; f[2] = a.z; f[3] = a.w; f[4] = b.x; f[5] = b.y; f[6] = b.z; f[7] = b.w;
  }
};

// Element stores for KV pools.
__device__ __forceinline__ void store_elem(float* p, float v) { *p = v; }
__device__ __forceinline__ void store_elem(bf16_t* p, float v) { *p = (bf16_t)f32_to_bf16(v); }
__device__ __forceinline__ float load_elem(const float* p) { return *p; }
__device__ __forceinline__ float load_elem(const bf16_t* p) { return bf16_to_f32(*p); }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, SSD_WAVE);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, SSD_WAVE));
  return v;
}

// (value, index) maximum; equal values resolve to the lower index.
__device__ __forceinline__ void argmax_merge(float& v, int& i, float v2, int i2) {
  if (v2 > v || (v2 == v && i2 < i)) { v = v2; i = i2; }
}

__device__ __forceinline__ void wave_argmax(float& v, int& i) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    float v2 = __shfl_xor(v, o, SSD_WAVE);
    int i2 = __shfl_xor(i, o, SSD_WAVE);
    argmax_merge(v, i, v2, i2);
  }
}

// tanh form of GELU (T5-v1.1 gated FFN, imitation network)
__device__ __forceinline__ float gelu_tanh(float u) {
  const float c = 0.7978845608028654f;  // sqrt(2/pi)
  return 0.5f * u * (1.0f + tanhf(c * (u + 0.044715f * u * u * u)));
}

__device__ __forceinline__ float silu(float u) { return u / (1.0f + expf(-u)); }
