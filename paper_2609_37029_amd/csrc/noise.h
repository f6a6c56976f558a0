// Counter-based noise shared by the sampler and the verifier: Philox4x64-10
// (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy as 1, 2, 3",
// SC 2011) keyed by (seed, step), a uniform made exactly from 23 of its bits,
// and Gumbel noise from a logarithm written as a fixed sequence of IEEE fp32
// operations, so that the noise is a pure function of (seed, step, counter).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ldr {

constexpr int kGroup = 8;  // tokens per Philox block (4 words of 64 bits)

constexpr uint64_t kM0 = 0xD2E7470EE14C6C93ull, kM1 = 0xCA5A826395121157ull;
constexpr uint64_t kW0 = 0x9E3779B97F4A7C15ull, kW1 = 0xBB67AE8584CAA73Bull;

// 128-bit product M x, M a constant: four 32 x 32 + 64 multiply-adds
// (v_mad_u64_u32), the middle column carried through p1 and p2.
template <uint64_t M>
__device__ inline void mulhilo(uint64_t x, uint64_t& hi, uint64_t& lo) {
  constexpr uint32_t Ml = (uint32_t)M, Mh = (uint32_t)(M >> 32);
  const uint32_t xl = (uint32_t)x, xh = (uint32_t)(x >> 32);
  const uint64_t p0 = (uint64_t)Ml * xl;
  const uint64_t p1 = (uint64_t)Mh * xl + (p0 >> 32);
  const uint64_t p2 = (uint64_t)Ml * xh + (uint32_t)p1;
  lo = (p2 << 32) | (uint32_t)p0;
  hi = (uint64_t)Mh * xh + (p1 >> 32) + (p2 >> 32);
}

__device__ inline void philox4x64_10(uint64_t c[4], uint64_t k0, uint64_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) { k0 += kW0; k1 += kW1; }
    uint64_t hi0, lo0, hi1, lo1;
    mulhilo<kM0>(c[0], hi0, lo0);
    mulhilo<kM1>(c[2], hi1, lo1);
    const uint64_t n0 = hi1 ^ c[1] ^ k0, n2 = hi0 ^ c[3] ^ k1;
    c[0] = n0; c[1] = lo1; c[2] = n2; c[3] = lo0;
  }
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

// The 8 noise words of tokens [8c, 8c+8) of `row` in counter stream `stream`
// (counter (c, row, stream, 0)).
__device__ inline void noise_group(uint64_t seed, uint64_t step, uint64_t row, uint64_t stream,
                                   uint64_t c, uint32_t out[kGroup]) {
  uint64_t w[4] = {c, row, stream, 0};
  philox4x64_10(w, seed, step);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    out[2 * i] = (uint32_t)w[i];
    out[2 * i + 1] = (uint32_t)(w[i] >> 32);
  }
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
