// Block-view attention on MFMA for bf16 views (Eq. 6; App. A.1; Sec. 2.4).
//
// One workgroup per (kv group g, sequence b), one wave per query head of the
// group. Keys and values are consumed in chunks of 32 under one online
// softmax:
//   chunk 0      the block's own k / v (B rows, q/k RMSNorm + RoPE applied in
//                the prologue from the QKV split-K partials);
//   chunks 1..   the recent window of layer j, staged through LDS once for all
//                heads of the group (K rows as stored, V transposed), the
//                next chunk fetched into registers while the current one is
//                consumed;
//   last         the head's R summary entries: keys G[j,h] (bf16), values
//                M[j,h] kept in fp32 and accumulated on the VALU.
// S = Q K^T and O += P V run on v_mfma_f32_16x16x32_bf16 (16 query rows per
// wave = the B <= 16 slots); P goes through a per-wave LDS tile to change
// from the C layout to the A layout.
#include "ldr_internal.h"

namespace ldr {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int KC = 32;  // keys per chunk
constexpr int QR = 16;  // query rows per wave (block slots, zero-padded)

__device__ inline float sum16(float v) {  // over the 16 lanes of a row group
  for (int off = 1; off < 16; off <<= 1) v += __shfl_xor(v, off);
  return v;
}
__device__ inline float max16(float v) {
  for (int off = 1; off < 16; off <<= 1) v = fmaxf(v, __shfl_xor(v, off));
  return v;
}
__device__ inline float sum64(float v) {
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
  return v;
}
__device__ inline bf16x8 frag(const uint16_t* p) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(p));
}
__device__ inline void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

template <int D, int REP>
__global__ void __launch_bounds__(64 * REP) attention_mfma_kernel(AttnArgs a) {
  constexpr int NT = 64 * REP;
  constexpr int LDQ = D + 8;   // bf16 row of the Q / K tiles (conflict-free 16-row reads)
  constexpr int LDV = KC + 8;  // bf16 row of the V^T / P tiles
  constexpr int HALF = D / 2, NDT = D / 16, KS = D / 32;
  constexpr int CH = KC * D / 8;              // 16-byte pieces of one chunk matrix
  constexpr int PL = (CH + NT - 1) / NT;
  __shared__ __attribute__((aligned(16))) uint16_t Qs[REP][QR * LDQ];
  __shared__ __attribute__((aligned(16))) uint16_t Ks[2][KC * LDQ];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[2][D * LDV];
  __shared__ __attribute__((aligned(16))) uint16_t Pt[REP][QR * LDV];

  const int g = blockIdx.x, b = blockIdx.y;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int h = g * REP + w;
  const int B = a.B;
  const long t = a.pos[b];
  const int nv = t < a.W ? (int)t : a.W;
  const int nwin = (nv + KC - 1) / KC;
  const uint8_t* seq = a.arena + (size_t)b * a.stride;
  const size_t gw = (size_t)(a.layer * a.hkv + g) * a.W * D;
  const uint16_t* Kw = reinterpret_cast<const uint16_t*>(seq + a.kw) + gw;
  const uint16_t* Vw = reinterpret_cast<const uint16_t*>(seq + a.vw) + gw;

  uint4 kreg[PL], vreg[PL];
  auto fetch = [&](int c) {  // window rows [c*KC, c*KC + KC) into registers
#pragma unroll
    for (int i = 0; i < PL; ++i) {
      const int idx = threadIdx.x + i * NT;
      const int r = idx / (D / 8), col = (idx % (D / 8)) * 8, slot = c * KC + r;
      if (idx < CH && slot < nv) {
        kreg[i] = *reinterpret_cast<const uint4*>(Kw + (size_t)slot * D + col);
        vreg[i] = *reinterpret_cast<const uint4*>(Vw + (size_t)slot * D + col);
      } else {
        kreg[i] = make_uint4(0, 0, 0, 0);
        vreg[i] = make_uint4(0, 0, 0, 0);
      }
    }
  };
  auto stash = [&](int buf) {  // K rows as they are, V transposed
#pragma unroll
    for (int i = 0; i < PL; ++i) {
      const int idx = threadIdx.x + i * NT;
      if (idx < CH) {
        const int r = idx / (D / 8), col = (idx % (D / 8)) * 8;
        *reinterpret_cast<uint4*>(&Ks[buf][r * LDQ + col]) = kreg[i];
        const uint16_t* v = reinterpret_cast<const uint16_t*>(&vreg[i]);
#pragma unroll
        for (int j = 0; j < 8; ++j) Vt[buf][(col + j) * LDV + r] = v[j];
      }
    }
  };
  if (nwin > 0) fetch(0);

  // ---- prologue: q rows of every head of the group, then block k and v rows.
  // One wave per row; lane e < d/2 holds the rotary pair (e, e + d/2). The
  // split-K partials of GROUP rows are loaded before any of them is reduced.
  constexpr int ROWS = (REP + 2) * QR, GROUP = 8;
  auto decode = [&](int r, int& kind, int& hh, int& i, int& col) {
    hh = 0;
    if (r < REP * QR) {
      kind = 0; hh = r / QR; i = r % QR; col = (g * REP + hh) * D;
    } else if (r < (REP + 1) * QR) {
      kind = 1; i = r - REP * QR; col = (a.hq + g) * D;
    } else {
      kind = 2; i = r - (REP + 1) * QR; col = (a.hq + a.hkv + g) * D;
    }
  };
  for (int base = w; base < ROWS; base += REP * GROUP) {
    float x1[GROUP], x2[GROUP];
#pragma unroll
    for (int k = 0; k < GROUP; ++k) {
      const int r = base + k * REP;
      x1[k] = 0.f;
      x2[k] = 0.f;
      int kind, hh, i, col;
      decode(r, kind, hh, i, col);
      if (r < ROWS && i < B && lane < HALF) {
        const float* src = a.part + ((long)b * B + i) * a.qkv_out + col;
        for (int s = 0; s < a.splits; ++s) {
          x1[k] += src[s * a.split_stride + lane];
          x2[k] += src[s * a.split_stride + lane + HALF];
        }
      }
    }
#pragma unroll
    for (int k = 0; k < GROUP; ++k) {
      const int r = base + k * REP;
      if (r >= ROWS) break;  // uniform across the wave
      int kind, hh, i, col;
      decode(r, kind, hh, i, col);
      const bool live = i < B && lane < HALF;
      const long m = (long)b * B + i;
      float y1 = x1[k], y2 = x2[k];
      if (kind != 2) {  // per-head RMSNorm, then rotate-half RoPE at position t + i
        const float inv = rsqrtf(sum64(y1 * y1 + y2 * y2) / D + a.eps);
        if (live) {
          const uint16_t* gain = static_cast<const uint16_t*>(kind == 0 ? a.q_norm : a.k_norm);
          const float z1 = y1 * inv * bf16_to_f32(gain[lane]);
          const float z2 = y2 * inv * bf16_to_f32(gain[lane + HALF]);
          const float cs = a.rope[m * HALF + lane];
          const float sn = a.rope[(long)a.M * HALF + m * HALF + lane];
          y1 = z1 * cs - z2 * sn;
          y2 = z1 * sn + z2 * cs;
        }
      }
      if (lane < HALF) {
        const uint16_t v1 = f32_to_bf16(y1), v2 = f32_to_bf16(y2);
        if (kind == 0) {
          Qs[hh][i * LDQ + lane] = v1; Qs[hh][i * LDQ + lane + HALF] = v2;
        } else if (kind == 1) {
          Ks[0][i * LDQ + lane] = v1; Ks[0][i * LDQ + lane + HALF] = v2;
        } else {
          Vt[0][lane * LDV + i] = v1; Vt[0][(lane + HALF) * LDV + i] = v2;
        }
      }
    }
  }
  for (int idx = threadIdx.x; idx < (KC - QR) * D; idx += NT) {  // padding keys of chunk 0
    const int r = QR + idx / D, e = idx % D;
    Ks[0][r * LDQ + e] = 0;
    Vt[0][e * LDV + r] = 0;
  }
  __syncthreads();

  bf16x8 qf[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) qf[kk] = frag(&Qs[w][(lane & 15) * LDQ + kk * 32 + (lane >> 4) * 8]);

  f32x4 o[NDT];
#pragma unroll
  for (int n = 0; n < NDT; ++n) o[n] = f32x4{0.f, 0.f, 0.f, 0.f};
  float mrow[4], lrow[4];  // rows (lane / 16) * 4 + v; lrow is this lane's partial sum
#pragma unroll
  for (int v = 0; v < 4; ++v) { mrow[v] = -INFINITY; lrow[v] = 0.f; }
  const float scale = a.inv_sqrt_d;

  // online softmax over a 32-key score tile sc (C layout), valid keys < nvalid
  auto absorb = [&](f32x4 (&sc)[2], int nvalid) {
    float cmax[4];
#pragma unroll
    for (int v = 0; v < 4; ++v) cmax[v] = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int key = kt * 16 + (lane & 15);
        const float s = key < nvalid ? sc[kt][v] * scale : -INFINITY;
        sc[kt][v] = s;
        cmax[v] = fmaxf(cmax[v], s);
      }
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const float mnew = fmaxf(mrow[v], max16(cmax[v]));
      const float alpha = __expf(mrow[v] - mnew);  // first tile: exp(-inf) = 0
      mrow[v] = mnew;
      lrow[v] *= alpha;
#pragma unroll
      for (int n = 0; n < NDT; ++n) o[n][v] *= alpha;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        const float p = __expf(sc[kt][v] - mnew);
        sc[kt][v] = p;
        lrow[v] += p;
      }
    }
  };

  for (int c = 0; c <= nwin; ++c) {
    const int buf = c & 1;
    if (c >= 1 && c < nwin) fetch(c);
    const int nvalid = c == 0 ? B : min(KC, nv - (c - 1) * KC);
    f32x4 sc[2];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      sc[kt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < KS; ++kk)
        sc[kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
            qf[kk], frag(&Ks[buf][(kt * 16 + (lane & 15)) * LDQ + kk * 32 + (lane >> 4) * 8]),
            sc[kt], 0, 0, 0);
    }
    absorb(sc, nvalid);
    // P: C layout -> per-wave LDS tile -> A layout
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int v = 0; v < 4; ++v)
        Pt[w][((lane >> 4) * 4 + v) * LDV + kt * 16 + (lane & 15)] = f32_to_bf16(sc[kt][v]);
    wave_lds_sync();
    const bf16x8 pf = frag(&Pt[w][(lane & 15) * LDV + (lane >> 4) * 8]);
#pragma unroll
    for (int n = 0; n < NDT; ++n)
      o[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
          pf, frag(&Vt[buf][(n * 16 + (lane & 15)) * LDV + (lane >> 4) * 8]), o[n], 0, 0, 0);
    wave_lds_sync();
    if (c < nwin) stash((c + 1) & 1);
    lds_barrier();
  }

  // ---- summary entries of head h: keys G[j,h] (bf16), values M[j,h] (fp32) ----
  if (t > 0) {
    const uint16_t* Gh = static_cast<const uint16_t*>(a.G) + ((size_t)(a.layer * a.hq + h) * a.R) * D;
    const float* Mh = reinterpret_cast<const float*>(seq + a.m_off) +
                      ((size_t)(a.layer * a.hq + h) * a.R) * D;
    f32x4 sc[2];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      sc[kt] = f32x4{0.f, 0.f, 0.f, 0.f};
      const int r = kt * 16 + (lane & 15);
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) {
        const bf16x8 gf = r < a.R ? frag(Gh + (size_t)r * D + kk * 32 + (lane >> 4) * 8)
                                  : __builtin_bit_cast(bf16x8, make_uint4(0, 0, 0, 0));
        sc[kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qf[kk], gf, sc[kt], 0, 0, 0);
      }
    }
    absorb(sc, a.R);
    for (int r = 0; r < a.R; ++r) {  // O[q][e] += p[q][r] M[r][e] in fp32
      const int src = (lane & 48) | (r & 15);
      float pr[4];
#pragma unroll
      for (int v = 0; v < 4; ++v) pr[v] = __shfl(r < 16 ? sc[0][v] : sc[1][v], src);
#pragma unroll
      for (int n = 0; n < NDT; ++n) {
        const float mv = Mh[(size_t)r * D + n * 16 + (lane & 15)];
#pragma unroll
        for (int v = 0; v < 4; ++v) o[n][v] += pr[v] * mv;
      }
    }
  }

  uint16_t* out = static_cast<uint16_t*>(a.o);
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int q = (lane >> 4) * 4 + v;
    const float inv = 1.f / sum16(lrow[v]);
    if (q < B) {
      uint16_t* row = out + ((long)b * B + q) * ((long)a.hq * D) + (long)h * D + (lane & 15);
#pragma unroll
      for (int n = 0; n < NDT; ++n) row[n * 16] = f32_to_bf16(o[n][v] * inv);
    }
  }
}

template <int D>
hipError_t launch_d(const AttnArgs& a, int hkv, int batch, hipStream_t st) {
  const dim3 grid(hkv, batch);
  switch (a.rep) {
    case 1: hipLaunchKernelGGL((attention_mfma_kernel<D, 1>), grid, dim3(64), 0, st, a); break;
    case 2: hipLaunchKernelGGL((attention_mfma_kernel<D, 2>), grid, dim3(128), 0, st, a); break;
    case 4: hipLaunchKernelGGL((attention_mfma_kernel<D, 4>), grid, dim3(256), 0, st, a); break;
    case 8: hipLaunchKernelGGL((attention_mfma_kernel<D, 8>), grid, dim3(512), 0, st, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

bool attention_mfma_supported(int d, int rep, int B, int R) {
  return (d == 64 || d == 128) && (rep == 1 || rep == 2 || rep == 4 || rep == 8) && B <= QR &&
         R <= 2 * 16;
}

hipError_t launch_attention_mfma(const AttnArgs& a, int hkv, int batch, hipStream_t st) {
  if (!attention_mfma_supported(a.d, a.rep, a.B, a.R)) return hipErrorInvalidValue;
  return a.d == 128 ? launch_d<128>(a, hkv, batch, st) : launch_d<64>(a, hkv, batch, st);
}

}  // namespace ldr
