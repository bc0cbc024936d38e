// Device helpers of the GSQ kernels: Philox4x32-10, the noise transforms, bf16 rounding.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gsq {

// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11): ten rounds, each multiplying words
// 0 and 2 by the round multipliers and mixing the 64-bit products' halves with the other
// words and the round key; the key advances by the two Weyl constants between rounds.
struct U4 { uint32_t x, y, z, w; };

__device__ __forceinline__ U4 philox10(U4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t p0 = (uint64_t)0xD2511F53u * c.x;
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * c.z;
    c = U4{(uint32_t)(p1 >> 32) ^ c.y ^ k0, (uint32_t)p1, (uint32_t)(p0 >> 32) ^ c.w ^ k1,
           (uint32_t)p0};
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return c;
}

// Noise layout: the four coordinates e0 .. e0+3 of an aligned chunk (e0 = e - e mod 4) read
// their 4K values, coordinate e0+q / level k at flat position f = q K + k, from K Philox calls:
// call j has counter (e0 mod 2^32, e0 >> 32, t, tag*256 + j) and position f takes word
// f mod 4 of call f div 4.  tag = sample*256 + stream, stream 0 = step noise, 1 = initial logit
// noise, sample = index of an independent draw within one step; key = seed.
__device__ __forceinline__ U4 noise_words(uint64_t seed, uint64_t e0, uint32_t t, uint32_t tag,
                                          uint32_t j) {
  return philox10(U4{(uint32_t)e0, (uint32_t)(e0 >> 32), t, tag * 256u + j}, (uint32_t)seed,
                  (uint32_t)(seed >> 32));
}

__device__ __forceinline__ uint32_t word_of(const U4& w, int r) {
  return r == 0 ? w.x : r == 1 ? w.y : r == 2 ? w.z : w.w;
}

// u = (top 23 bits + 1/2) * 2^-23, exact in fp32, in [2^-24, 1 - 2^-24]: the float with
// mantissa m = x >> 9 and exponent 0 is 1 + m 2^-23; subtracting 1 - 2^-24 (exact, the result
// has at most 24 significant bits) leaves (m + 1/2) 2^-23.
__device__ __forceinline__ float uniform01(uint32_t x) {
  return __uint_as_float((x >> 9) | 0x3F800000u) - 0x1.fffffep-1f;
}

// Gumbel(0,1) sample -ln(-ln u): evaluated in fp64 and rounded once to fp32.
__device__ __forceinline__ float gumbel_exact(uint32_t x) {
  const double u = (double)uniform01(x);
  return (float)(-log(-log(u)));
}

// Gumbel(0,1) sample with the hardware base-2 logarithm:
// -ln(-ln u) = -ln2 * log2(-ln2 * log2 u).
__device__ __forceinline__ float gumbel_fast(uint32_t x) {
  constexpr float kLn2 = 0.69314718055994531f;
  const float u = uniform01(x);
  const float nl = __builtin_amdgcn_logf(u) * -kLn2;   // -ln u > 0
  return __builtin_amdgcn_logf(nl) * -kLn2;
}

// Logistic(0,1) sample ln u - ln(1 - u), the noise of a two-value relaxation with logits
// {-l, l}: its softmax sees the two Gumbel values only through their difference, which has this
// law.  1 - u is exact in fp32 (u has at most 24 significant bits below 1).  Exact: evaluated in
// fp64 and rounded once to fp32; fast: ln2 (log2 u - log2(1 - u)) with the hardware logarithm.
__device__ __forceinline__ float logistic_exact(uint32_t x) {
  const float u = uniform01(x);
  return (float)(log((double)u) - log((double)(1.0f - u)));
}

__device__ __forceinline__ float logistic_fast(uint32_t x) {
  constexpr float kLn2 = 0.69314718055994531f;
  const float u = uniform01(x);
  return (__builtin_amdgcn_logf(u) - __builtin_amdgcn_logf(1.0f - u)) * kLn2;
}

// Transform of a noise word: Gumbel values for categoricals, logistic values for binary pairs.
enum NoiseKind { kGumbel = 0, kLogistic = 1 };

template <int kKind, bool kExact>
__device__ __forceinline__ float noise_value(uint32_t x) {
  if constexpr (kKind == kLogistic) {
    if constexpr (kExact) return logistic_exact(x); else return logistic_fast(x);
  } else {
    if constexpr (kExact) return gumbel_exact(x); else return gumbel_fast(x);
  }
}

// The 4 x K noise values of the chunk starting at e0 (a multiple of 4) at step t.
template <int K, bool kExact, int kKind = kGumbel>
__device__ __forceinline__ void draw_chunk(float (&g)[4][K], uint64_t seed, uint64_t e0, uint32_t t,
                                           uint32_t sample) {
#pragma unroll
  for (int j = 0; j < K; ++j) {
    const U4 w = noise_words(seed, e0, t, sample * 256u, (uint32_t)j);
#pragma unroll
    for (int r = 0; r < 4; ++r)
      g[(4 * j + r) / K][(4 * j + r) % K] = noise_value<kKind, kExact>(word_of(w, r));
  }
}

// The K noise values of one coordinate e at step t (any e; draws only the calls it needs).
template <int K, bool kExact, int kKind = kGumbel>
__device__ __forceinline__ void draw_one(float (&g)[K], uint64_t seed, uint64_t e, uint32_t t) {
  const uint64_t e0 = e & ~(uint64_t)3;
  const int q = (int)(e & 3);
#pragma unroll
  for (int k = 0; k < K; ++k) {
    const int f = q * K + k;
    g[k] = noise_value<kKind, kExact>(word_of(noise_words(seed, e0, t, 0u, (uint32_t)(f >> 2)), f & 3));
  }
}

// float -> bf16 bits, round to nearest even (finite inputs).
__device__ __forceinline__ uint16_t bf16_rne(float f) {
  uint32_t b = __float_as_uint(f);
  b += 0x7FFFu + ((b >> 16) & 1u);
  return (uint16_t)(b >> 16);
}
__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

}  // namespace gsq
