// Device helpers shared by the kernels of the draft step (included by the HIP sources of
// the library only): vector types, bf16 / fp16 conversions and hi/lo splits, MFMA wrappers,
// write-through stores and coherent loads, and the MFMA A-fragment layout of activations.
#pragma once

#include "dflare_impl.h"

namespace dflare {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

#define GLOBAL __attribute__((address_space(1)))
#define CONSTANT __attribute__((address_space(4)))
#define LDSP __attribute__((address_space(3)))

constexpr int kLdsBytes = 160 * 1024;

__device__ __forceinline__ float bf2f(uint32_t b) { return __uint_as_float(b << 16); }

// float -> bf16 bits, round to nearest even (inputs are finite).
__device__ __forceinline__ uint32_t f2bf(float x) {
  uint32_t u = __float_as_uint(x);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

__device__ __forceinline__ void split_pack8(const float* v, u32x4& hi, u32x4& lo) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    uint32_t h0 = f2bf(v[2 * e]), h1 = f2bf(v[2 * e + 1]);
    uint32_t l0 = f2bf(v[2 * e] - bf2f(h0)), l1 = f2bf(v[2 * e + 1] - bf2f(h1));
    hi[e] = h0 | (h1 << 16);
    lo[e] = l0 | (l1 << 16);
  }
}

__device__ __forceinline__ f32x4 mfma(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mfma_h(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a),
                                                __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
}

// float -> fp16 bits, round to nearest even, saturated to +-65504 (the KV cache format)
__device__ __forceinline__ uint16_t f2h(float x) {
  return __builtin_bit_cast(uint16_t, (_Float16)fminf(fmaxf(x, -65504.f), 65504.f));
}
__device__ __forceinline__ float h2f(uint32_t b) { return (float)__builtin_bit_cast(_Float16, (uint16_t)b); }

// fp16 hi/lo split of 8 values inside the fp16 range (attention probabilities): hi rounded
// toward zero by the packed two-value conversion, lo = x - hi (exact in fp32) converted the same
// way; hi + lo keeps about 21 significant bits
__device__ __forceinline__ void split_pack8_hz(const float* v, u32x4& hi, u32x4& lo) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const auto h = __builtin_amdgcn_cvt_pkrtz(v[2 * e], v[2 * e + 1]);
    const auto l = __builtin_amdgcn_cvt_pkrtz(v[2 * e] - (float)h[0], v[2 * e + 1] - (float)h[1]);
    hi[e] = __builtin_bit_cast(uint32_t, h);
    lo[e] = __builtin_bit_cast(uint32_t, l);
  }
}

// fp16 hi/lo split of 8 floats (x ~= hi + lo with about 22 significant bits)
__device__ __forceinline__ void split_pack8_h(const float* v, u32x4& hi, u32x4& lo) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const uint32_t h0 = f2h(v[2 * e]), h1 = f2h(v[2 * e + 1]);
    const uint32_t l0 = f2h(v[2 * e] - h2f(h0)), l1 = f2h(v[2 * e + 1] - h2f(h1));
    hi[e] = h0 | (h1 << 16);
    lo[e] = l0 | (l1 << 16);
  }
}

// Every buffer lives in device (global) memory; pointers that come from memory rather than
// from kernel arguments are cast to the global address space so that the compiler emits
// global rather than flat memory instructions.
template <typename T>
__device__ __forceinline__ GLOBAL T* gbl(T* p) {
  return (GLOBAL T*)p;
}
template <typename T>
__device__ __forceinline__ const GLOBAL T* gbl(const T* p) {
  return (const GLOBAL T*)p;
}

// ---- write-through stores and coherent loads ----
__device__ __forceinline__ void st_wt(float* p, float v) {
  __hip_atomic_store(gbl(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_wt(uint32_t* p, uint32_t v) {
  __hip_atomic_store(gbl(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_wt(int* p, int v) {
  __hip_atomic_store(gbl(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_wt(uint16_t* p, uint16_t v) {
  __hip_atomic_store(gbl(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_wt8(void* p, uint64_t v) {
  __hip_atomic_store(gbl(reinterpret_cast<uint64_t*>(p)), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_wt16(void* p, u32x4 v) {
  uint64_t* q = reinterpret_cast<uint64_t*>(p);
  st_wt8(q, (uint64_t)v[0] | ((uint64_t)v[1] << 32));
  st_wt8(q + 1, (uint64_t)v[2] | ((uint64_t)v[3] << 32));
}
__device__ __forceinline__ float ld_coh(const float* p) {
  return __hip_atomic_load(gbl(const_cast<float*>(p)), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int ld_coh(const int* p) {
  return __hip_atomic_load(gbl(const_cast<int*>(p)), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float2 ld_coh2(const void* p) {
  const uint64_t v = __hip_atomic_load(gbl(reinterpret_cast<uint64_t*>(const_cast<void*>(p))), __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
  return make_float2(__uint_as_float((uint32_t)v), __uint_as_float((uint32_t)(v >> 32)));
}
// 16-byte coherent load (two 8-byte agent-scope loads)
__device__ __forceinline__ f32x4 ld_coh16(const f32x4* p) {
  const float2 x = ld_coh2(p), y = ld_coh2(reinterpret_cast<const float*>(p) + 2);
  return f32x4{x.x, x.y, y.x, y.y};
}
// an integer the compiler cannot see through (keeps address arithmetic where it is written)
__device__ __forceinline__ int opaque(int x) {
  asm volatile("" : "+v"(x));
  return x;
}

// wait until this wave's memory operations (stores included) have completed
__device__ __forceinline__ void wait_vm() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// ---- temperature sampling: Gumbel-max draws ----
// Philox4x64-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy as 1, 2, 3",
// SC 2011) of the counter (c0, c1, c2, c3) under the key (k0, k1); the four output words
// replace the counter.
__device__ __forceinline__ void philox4x64_10(uint64_t& c0, uint64_t& c1, uint64_t& c2, uint64_t& c3, uint64_t k0,
                                              uint64_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t hi0 = __umul64hi(c0, 0xD2E7470EE14C6C93ull), lo0 = c0 * 0xD2E7470EE14C6C93ull;
    const uint64_t hi1 = __umul64hi(c2, 0xCA5A826395121157ull), lo1 = c2 * 0xCA5A826395121157ull;
    c0 = hi1 ^ c1 ^ k0;
    c1 = lo1;
    c2 = hi0 ^ c3 ^ k1;
    c3 = lo0;
    k0 += 0x9E3779B97F4A7C15ull;
    k1 += 0xBB67AE8584CAA73Bull;
  }
}

// Temperature sampling draws token argmax_v (z_v / T + G_v), a draw from softmax(z / T), with
// Gumbel noise G = -log(-log U).  U of vocabulary id v at block position b, in draft call
// `draw` of sequence slot `slot`, comes from output word b % 4 of Philox4x64-10 at counter
// (v, b / 4, draw, slot) under key (seed, 0): one call serves four consecutive positions.
// gumbel_of_word: U = (top 23 bits of the word + 1/2) / 2^23, exact in fp32 and at most
// 1 - 2^-24, so the noise is finite.
__device__ __forceinline__ float gumbel_of_word(uint64_t x) {
  const float u = ((float)(uint32_t)(x >> 41) + 0.5f) * 1.1920928955078125e-7f;  // 2^-23
  return -logf(-logf(u));
}

// the four Philox words of counter (v, q, draw, slot): the noise words of positions 4 q .. 4 q + 3
__device__ __forceinline__ void gumbel_words(unsigned long long seed, int v, int q, unsigned draw, int slot,
                                             uint64_t w[4]) {
  w[0] = (uint64_t)v;
  w[1] = (uint64_t)q;
  w[2] = (uint64_t)draw;
  w[3] = (uint64_t)slot;
  philox4x64_10(w[0], w[1], w[2], w[3], seed, 0ull);
}

// the noise of positions 4 q .. 4 q + 3 (one Philox call)
__device__ __forceinline__ void gumbel_noise4(unsigned long long seed, int v, int q, unsigned draw, int slot,
                                              float out[4]) {
  uint64_t c0 = (uint64_t)v, c1 = (uint64_t)q, c2 = (uint64_t)draw, c3 = (uint64_t)slot;
  philox4x64_10(c0, c1, c2, c3, seed, 0ull);
  out[0] = gumbel_of_word(c0);
  out[1] = gumbel_of_word(c1);
  out[2] = gumbel_of_word(c2);
  out[3] = gumbel_of_word(c3);
}

// the noise of one position b
__device__ __forceinline__ float gumbel_noise1(unsigned long long seed, int v, int b, unsigned draw, int slot) {
  uint64_t c0 = (uint64_t)v, c1 = (uint64_t)(b >> 2), c2 = (uint64_t)draw, c3 = (uint64_t)slot;
  philox4x64_10(c0, c1, c2, c3, seed, 0ull);
  const int k = b & 3;
  return gumbel_of_word(k == 0 ? c0 : k == 1 ? c1 : k == 2 ? c2 : c3);
}

// Activations handed from one GEMM to the next are stored directly in the A-operand
// layout of v_mfma_f32_16x16x32_bf16, as two bf16 planes hi and lo (x ~= hi + lo):
//   element (row, k) of a [rows, K] matrix sits in 16-row tile row/16, k-tile k/32,
//   lane (row % 16) + 16 * ((k % 32) / 8), slot k % 8; a (row-tile, k-tile) is 1 KiB.
__device__ __forceinline__ long frag_off(int row, int k, int Kt) {
  return ((((long)(row >> 4) * Kt + (k >> 5)) * 64 + (row & 15) + ((k & 31) >> 3) * 16) << 3) + (k & 7);
}

// hi/lo planes of two consecutive elements (k even), one 32-bit word per plane
__device__ __forceinline__ void frag_pair(float v0, float v1, uint32_t& hi, uint32_t& lo) {
  const uint32_t h0 = f2bf(v0), h1 = f2bf(v1);
  hi = h0 | (h1 << 16);
  lo = f2bf(v0 - bf2f(h0)) | (f2bf(v1 - bf2f(h1)) << 16);
}
__device__ __forceinline__ void store_frag_pair(uint32_t* hi, uint32_t* lo, int row, int k, int Kt, float v0,
                                                float v1) {
  uint32_t h, l;
  frag_pair(v0, v1, h, l);
  const long o = frag_off(row, k, Kt) >> 1;
  hi[o] = h;
  lo[o] = l;
}
__device__ __forceinline__ void store_frag_pair_wt(uint32_t* hi, uint32_t* lo, int row, int k, int Kt, float v0,
                                                   float v1) {
  uint32_t h, l;
  frag_pair(v0, v1, h, l);
  const long o = frag_off(row, k, Kt) >> 1;
  st_wt(hi + o, h);
  st_wt(lo + o, l);
}

}  // namespace dflare
