// Counter-based noise shared by the sampler and the verifier: Philox4x32-10
// (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy as 1, 2, 3",
// SC 2011) keyed by the seed, a uniform made exactly from 23 of its bits, and
// Gumbel noise from a logarithm written as a fixed sequence of IEEE fp32
// operations, so that the noise is a pure function of (seed, step, stream,
// row, token). Token v of row r in stream s is word v mod 4 of the block of
// counter (v div 4, r, step mod 2^32, (step div 2^32) mod 2^30 + 2^30 s), key
// (seed mod 2^32, seed div 2^32). The 32-bit variant gives each 32 x 32-bit
// product (one v_mad_u64_u32) 32 output bits, twice the 64-bit variant's.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ldr {

constexpr int kGroup = 8;  // tokens per noise group: two Philox blocks of 4 words

constexpr uint32_t kM0 = 0xD2511F53u, kM1 = 0xCD9E8D57u;   // multipliers
constexpr uint32_t kW0 = 0x9E3779B9u, kW1 = 0xBB67AE85u;   // Weyl key increments

__device__ inline void philox4x32_10(uint32_t c[4], uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) { k0 += kW0; k1 += kW1; }
    const uint64_t p0 = (uint64_t)kM0 * c[0], p1 = (uint64_t)kM1 * c[2];
    const uint32_t n0 = (uint32_t)(p1 >> 32) ^ c[1] ^ k0;
    const uint32_t n2 = (uint32_t)(p0 >> 32) ^ c[3] ^ k1;
    c[0] = n0; c[1] = (uint32_t)p1; c[2] = n2; c[3] = (uint32_t)p0;
  }
}

// Key words and the two upper counter words of a (seed, step, stream).
struct NoiseKey { uint32_t k0, k1, c2, c3; };
__device__ inline NoiseKey noise_key(uint64_t seed, uint64_t step, uint32_t stream) {
  return NoiseKey{(uint32_t)seed, (uint32_t)(seed >> 32), (uint32_t)step,
                  ((uint32_t)(step >> 32) & 0x3FFFFFFFu) | (stream << 30)};
}

// The 4 words of block `blk` (tokens 4 blk .. 4 blk + 3) of `row`.
__device__ inline void noise_block(const NoiseKey& k, uint32_t row, uint32_t blk,
                                   uint32_t out[4]) {
  uint32_t c[4] = {blk, row, k.c2, k.c3};
  philox4x32_10(c, k.k0, k.k1);
#pragma unroll
  for (int i = 0; i < 4; ++i) out[i] = c[i];
}

// Natural log of a positive normal float: x = 2^e m, m folded into
// (sqrt(1/2), sqrt(2)], log x = e ln2 + 2 atanh(f), f = (m-1)/(m+1), with the
// odd series of atanh to f^11. Each operation is one IEEE fp32 rounding.
__device__ inline float fixed_logf(float x) {
#pragma clang fp contract(off)
  const float kC3 = __uint_as_float(0x3EAAAAABu), kC5 = __uint_as_float(0x3E4CCCCDu);
  const float kC7 = __uint_as_float(0x3E124925u), kC9 = __uint_as_float(0x3DE38E39u);
  const float kC11 = __uint_as_float(0x3DBA2E8Cu);
  const float kLn2Hi = __uint_as_float(0x3F317200u), kLn2Lo = __uint_as_float(0x35BFBE8Eu);
  const float kSqrt2 = __uint_as_float(0x3FB504F3u);
  const uint32_t bits = __float_as_uint(x);
  int e = (int)((bits >> 23) & 0xffu) - 127;
  float m = __uint_as_float((bits & 0x7fffffu) | 0x3f800000u);
  if (m > kSqrt2) { m = m * 0.5f; e += 1; }
  const float ef = (float)e;
  const float f = (m - 1.0f) / (m + 1.0f);
  const float s = f * f;
  float p = kC11;
  p = p * s + kC9;
  p = p * s + kC7;
  p = p * s + kC5;
  p = p * s + kC3;
  p = p * s + 1.0f;
  const float r = (f * 2.0f) * p;
  const float lo = ef * kLn2Lo + r;
  return ef * kLn2Hi + lo;
}

// u = (2 (bits >> 9) + 1) 2^-24: exact in fp32, strictly inside (0, 1).
__device__ inline float uniform_from_bits(uint32_t bits) {
#pragma clang fp contract(off)
  return ((float)(bits >> 9) * 2.0f + 1.0f) * 5.9604644775390625e-08f;  // 2^-24
}

__device__ inline float gumbel_from_bits(uint32_t bits) {
  return -fixed_logf(-fixed_logf(uniform_from_bits(bits)));
}

// The noise words of tokens [G g, G g + G) of `row` in stream `stream` (G a
// multiple of 4: Philox blocks G / 4 g .. + G / 4, one word per token).
template <int G>
__device__ inline void noise_group(uint64_t seed, uint64_t step, uint64_t row, uint32_t stream,
                                   uint64_t g, uint32_t (&out)[G]) {
  static_assert(G % 4 == 0, "whole Philox blocks");
  const NoiseKey k = noise_key(seed, step, stream);
#pragma unroll
  for (int b = 0; b < G / 4; ++b)
    noise_block(k, (uint32_t)row, (uint32_t)((G / 4) * g + b), out + 4 * b);
}

// Upper bound of the Gumbel noise g = -log(-log u) of 23-bit uniform index k,
// u = (2k + 1) 2^-24, from integer arithmetic: -log u >= 1 - u = n 2^-24 with
// n = 2^24 - 1 - 2k, so g <= 24 ln2 - ln n, and ln n >= ln2 (e + m - 1) for
// n = m 2^e, m in [1, 2) (log2 m >= m - 1 on [1, 2]).
__device__ inline float gumbel_upper(uint32_t bits) {
  const uint32_t n = 0xFFFFFFu - 2u * (bits >> 9);
  const uint32_t nb = __float_as_uint((float)n);  // exact: n < 2^24
  const float e = (float)((int)(nb >> 23) - 127);
  const float m = __uint_as_float((nb & 0x7FFFFFu) | 0x3F800000u);
  return __uint_as_float(0x3F317218u) * (25.0f - e - m);  // ln2 rounded up
}

}  // namespace ldr
