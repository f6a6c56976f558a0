// Block-view attention on MFMA for bf16 views (Eq. 6; App. A.1; Sec. 2.4).
//
// One workgroup per (kv group g, sequence b) and up to 4 query heads of the
// group, one wave per head. Keys and values are consumed in chunks of 32 under
// one online softmax:
//   chunk 0      the block's own k / v (B rows, normalised and rotated by the
//                QKV finishing kernel);
//   chunks 1..   the recent window of layer j, staged through LDS once for all
//                heads of the group (K rows and the transposed V rows as
//                stored in the views), the next chunks fetched into
//                registers while the current one is consumed;
//   last         the head's R summary entries: keys G[j,h] (bf16), values
//                M[j,h] kept in fp32 and accumulated on the VALU; both are
//                loaded at the start and parked in LDS after the prologue.
// S = Q K^T and O += P V run on v_mfma_f32_16x16x32_bf16 (16 query rows per
// wave = the B <= 16 slots); P goes through a per-wave LDS tile to change
// from the C layout to the A layout.
#include "ldr_internal.h"

namespace ldr {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

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

// HPW query heads of one kv group per workgroup (a group with more heads
// spreads over rep / HPW workgroups, each reading the group's window).
template <int D, int HPW>
__global__ void __launch_bounds__(64 * HPW) attention_mfma_kernel(AttnArgs a) {
  constexpr int NT = 64 * HPW;
  constexpr int LDQ = D + 8;   // bf16 row of the Q / K tiles (conflict-free 16-row reads)
  constexpr int LDV = KC + 8;  // bf16 row of the V^T / P tiles
  constexpr int NDT = D / 16, KS = D / 32;
  constexpr int CH = KC * D / 8;              // 16-byte pieces of one chunk matrix
  constexpr int PL = (CH + NT - 1) / NT;
  __shared__ __attribute__((aligned(16))) uint16_t Qs[HPW][QR * LDQ];
  __shared__ __attribute__((aligned(16))) uint16_t Ks[2][KC * LDQ];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[2][D * LDV];
  __shared__ __attribute__((aligned(16))) uint16_t Pt[HPW][QR * LDV];
  // summary entries of the workgroup's heads: keys G (bf16), values M (fp32)
  constexpr int RMAX = 16;
  __shared__ __attribute__((aligned(16))) uint16_t Gs[HPW][RMAX * LDQ];
  __shared__ __attribute__((aligned(16))) float Ms[HPW][RMAX * D];

  const int per_group = a.rep / HPW;
  const int g = blockIdx.x / per_group, b = blockIdx.y;
  const int h0 = g * a.rep + (blockIdx.x % per_group) * HPW;  // first head of the workgroup
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int h = h0 + w;
  const int B = a.B;
  const long t = a.pos[b];
  const int nv = t < a.W ? (int)t : a.W;
  const int nwin = (nv + KC - 1) / KC;
  const uint8_t* seq = a.arena + (size_t)b * a.stride;
  const size_t gw = (size_t)(a.layer * a.hkv + g) * a.W * D;
  const uint16_t* Kw = reinterpret_cast<const uint16_t*>(seq + a.kw) + gw;
  const uint16_t* Vw = reinterpret_cast<const uint16_t*>(seq + a.vw) + gw;

  // Window chunks in flight: wk[p] / wv[p] hold chunk c + p while chunk c is
  // consumed (a ring of depth WD rotated by shifting). Fetches past the valid
  // rows reload the last valid row: its scores are masked.
  constexpr int WD = 3;
  u32x4 wk[WD][PL], wv[WD][PL];
#define LDR_FETCH(p, c)                                                                  \
  _Pragma("unroll") for (int i = 0; i < PL; ++i) {                                       \
    const int idx_ = (threadIdx.x + i * NT) % CH;                                        \
    const int slot_ = min((c) * KC + idx_ / (D / 8), nv - 1), col_ = (idx_ % (D / 8)) * 8; \
    wk[p][i] = *reinterpret_cast<const u32x4*>(Kw + (size_t)slot_ * D + col_);         \
    wv[p][i] = *reinterpret_cast<const u32x4*>(Vw + (size_t)(idx_ >> 2) * a.W +         \
                                               (c) * KC + (idx_ & 3) * 8);               \
  }
  if (nwin > 0) {
#pragma unroll
    for (int p = 0; p < WD; ++p) { LDR_FETCH(p, min(p, nwin - 1)) }
  }

  // Summary keys and values of the group's heads, loaded now (the prologue
  // hides their latency) and parked in LDS after it. Rows past R are zero.
  constexpr int SG = HPW * RMAX * D / 8;      // 16-byte pieces of G (bf16)
  constexpr int SM = HPW * RMAX * D / 4;      // 16-byte pieces of M (fp32)
  constexpr int GL = (SG + NT - 1) / NT, ML = (SM + NT - 1) / NT;
  uint4 greg[GL], mreg[ML];
  {
    const size_t hrow = (size_t)(a.layer * a.hq + h0) * a.R;  // first row of the workgroup
    const uint16_t* Gg = static_cast<const uint16_t*>(a.G) + hrow * D;
    const float* Mg = reinterpret_cast<const float*>(seq + a.m_off) + hrow * D;
#pragma unroll
    for (int i = 0; i < GL; ++i) {
      const int idx = threadIdx.x + i * NT;
      const int hh = idx / (RMAX * D / 8), r = (idx / (D / 8)) % RMAX, col = (idx % (D / 8)) * 8;
      greg[i] = (idx < SG && r < a.R && t > 0)
                    ? *reinterpret_cast<const uint4*>(Gg + ((size_t)hh * a.R + r) * D + col)
                    : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < ML; ++i) {
      const int idx = threadIdx.x + i * NT;
      const int hh = idx / (RMAX * D / 4), r = (idx / (D / 4)) % RMAX, col = (idx % (D / 4)) * 4;
      mreg[i] = (idx < SM && r < a.R && t > 0)
                    ? *reinterpret_cast<const uint4*>(Mg + ((size_t)hh * a.R + r) * D + col)
                    : make_uint4(0, 0, 0, 0);
    }
  }

  // ---- block rows: q of the workgroup's heads, k and v of the group (already
  // normalised and rotated), zero past the B slots of the 16-row tile.
  constexpr int QP = HPW * QR * D / 8, KP = QR * D / 8;  // 16-byte pieces
  constexpr int NP = QP + 2 * KP, PP = (NP + NT - 1) / NT;
  const uint16_t* qkv = static_cast<const uint16_t*>(a.qkv) + (size_t)b * B * a.qkv_out;
  u32x4 pre[PP];
#pragma unroll
  for (int i = 0; i < PP; ++i) {
    const int idx = threadIdx.x + i * NT;
    const int j = idx < QP ? idx % (QR * D / 8) : (idx - QP) % KP;
    const int row = j / (D / 8), c8 = (j % (D / 8)) * 8;
    const int col = idx < QP ? (h0 + idx / (QR * D / 8)) * D + c8
                  : idx < QP + KP ? (a.hq + g) * D + c8 : (a.hq + a.hkv + g) * D + c8;
    pre[i] = (idx < NP && row < B)
                 ? *reinterpret_cast<const u32x4*>(qkv + (size_t)row * a.qkv_out + col)
                 : u32x4{0u, 0u, 0u, 0u};
  }
#pragma unroll
  for (int i = 0; i < PP; ++i) {
    const int idx = threadIdx.x + i * NT;
    if (idx >= NP) break;
    const int j = idx < QP ? idx % (QR * D / 8) : (idx - QP) % KP;
    const int row = j / (D / 8), c8 = (j % (D / 8)) * 8;
    if (idx < QP) {
      *reinterpret_cast<u32x4*>(&Qs[idx / (QR * D / 8)][row * LDQ + c8]) = pre[i];
    } else if (idx < QP + KP) {
      *reinterpret_cast<u32x4*>(&Ks[0][row * LDQ + c8]) = pre[i];
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        Vt[0][(c8 + 2 * e) * LDV + row] = (uint16_t)(pre[i][e] & 0xffffu);
        Vt[0][(c8 + 2 * e + 1) * LDV + row] = (uint16_t)(pre[i][e] >> 16);
      }
    }
  }
  for (int idx = threadIdx.x; idx < (KC - QR) * D; idx += NT) {  // padding keys of chunk 0
    const int r = QR + idx / D, e = idx % D;
    Ks[0][r * LDQ + e] = 0;
    Vt[0][e * LDV + r] = 0;
  }
#pragma unroll
  for (int i = 0; i < GL; ++i) {
    const int idx = threadIdx.x + i * NT;
    if (idx < SG) {
      const int hh = idx / (RMAX * D / 8), r = (idx / (D / 8)) % RMAX, col = (idx % (D / 8)) * 8;
      *reinterpret_cast<uint4*>(&Gs[hh][r * LDQ + col]) = greg[i];
    }
  }
#pragma unroll
  for (int i = 0; i < ML; ++i) {
    const int idx = threadIdx.x + i * NT;
    if (idx < SM) {
      const int hh = idx / (RMAX * D / 4), r = (idx / (D / 4)) % RMAX, col = (idx % (D / 4)) * 4;
      *reinterpret_cast<uint4*>(&Ms[hh][r * D + col]) = mreg[i];
    }
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

  // Scores of one 32-key chunk in LDS buffer `buf`, the online softmax, and
  // O += P V on the same chunk.
#define LDR_CHUNK(buf, nvalid)                                                           \
  {                                                                                      \
    f32x4 sc[2];                                                                         \
    _Pragma("unroll") for (int kt = 0; kt < 2; ++kt) {                                   \
      sc[kt] = f32x4{0.f, 0.f, 0.f, 0.f};                                                \
      _Pragma("unroll") for (int kk = 0; kk < KS; ++kk) sc[kt] =                         \
          __builtin_amdgcn_mfma_f32_16x16x32_bf16(                                       \
              qf[kk], frag(&Ks[buf][(kt * 16 + (lane & 15)) * LDQ + kk * 32 + (lane >> 4) * 8]), \
              sc[kt], 0, 0, 0);                                                          \
    }                                                                                    \
    absorb(sc, nvalid);                                                                  \
    _Pragma("unroll") for (int kt = 0; kt < 2; ++kt)                                     \
        _Pragma("unroll") for (int v = 0; v < 4; ++v)                                    \
            Pt[w][((lane >> 4) * 4 + v) * LDV + kt * 16 + (lane & 15)] = f32_to_bf16(sc[kt][v]); \
    wave_lds_sync();                                                                     \
    const bf16x8 pf = frag(&Pt[w][(lane & 15) * LDV + (lane >> 4) * 8]);                 \
    _Pragma("unroll") for (int n = 0; n < NDT; ++n) o[n] =                               \
        __builtin_amdgcn_mfma_f32_16x16x32_bf16(                                         \
            pf, frag(&Vt[buf][(n * 16 + (lane & 15)) * LDV + (lane >> 4) * 8]), o[n], 0, 0, 0); \
    wave_lds_sync();                                                                     \
  }
  // K rows as they are; V^T rows (dim e, 32 keys) as stored, from ring slot 0
#define LDR_STASH(buf)                                                                   \
  _Pragma("unroll") for (int i = 0; i < PL; ++i) {                                       \
    const int idx_ = (threadIdx.x + i * NT) % CH;                                        \
    const int r_ = idx_ / (D / 8), col_ = (idx_ % (D / 8)) * 8;                          \
    *reinterpret_cast<u32x4*>(&Ks[buf][r_ * LDQ + col_]) = wk[0][i];                     \
    *reinterpret_cast<u32x4*>(&Vt[buf][(idx_ >> 2) * LDV + (idx_ & 3) * 8]) = wv[0][i];  \
  }

  if (nwin == 0) {
    LDR_CHUNK(0, B)
  } else {
    // chunk 0 is the block; chunk c >= 1 is window chunk c - 1 (LDS buffer c & 1)
    for (int c = 0; c <= nwin; ++c) {
      const int buf = c & 1;
      LDR_CHUNK(buf, c == 0 ? B : min(KC, nv - (c - 1) * KC))
      LDR_STASH(buf ^ 1)  // window chunk c (past the end: never read)
#pragma unroll
      for (int p = 0; p + 1 < WD; ++p)
#pragma unroll
        for (int i = 0; i < PL; ++i) {
          wk[p][i] = wk[p + 1][i];
          wv[p][i] = wv[p + 1][i];
        }
      LDR_FETCH(WD - 1, min(c + WD, nwin - 1))
      lds_barrier();
    }
  }
#undef LDR_STASH
#undef LDR_CHUNK
#undef LDR_FETCH

  // ---- summary entries of head h: keys G[j,h] (bf16), values M[j,h] (fp32) ----
  if (t > 0) {
    f32x4 sc[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};  // keys >= 16 masked
#pragma unroll
    for (int kk = 0; kk < KS; ++kk)
      sc[0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
          qf[kk], frag(&Gs[w][(lane & 15) * LDQ + kk * 32 + (lane >> 4) * 8]), sc[0], 0, 0, 0);
    absorb(sc, a.R);
    for (int r = 0; r < a.R; ++r) {  // O[q][e] += p[q][r] M[r][e] in fp32
      const int src = (lane & 48) | (r & 15);
      float pr[4];
#pragma unroll
      for (int v = 0; v < 4; ++v) pr[v] = __shfl(sc[0][v], src);
#pragma unroll
      for (int n = 0; n < NDT; ++n) {
        const float mv = Ms[w][r * D + n * 16 + (lane & 15)];
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
  const int hpw = a.rep < 4 ? a.rep : 4;
  const dim3 grid(hkv * (a.rep / hpw), batch);
  switch (hpw) {
    case 1: hipLaunchKernelGGL((attention_mfma_kernel<D, 1>), grid, dim3(64), 0, st, a); break;
    case 2: hipLaunchKernelGGL((attention_mfma_kernel<D, 2>), grid, dim3(128), 0, st, a); break;
    default: hipLaunchKernelGGL((attention_mfma_kernel<D, 4>), grid, dim3(256), 0, st, a); break;
  }
  return hipGetLastError();
}

}  // namespace

bool attention_mfma_supported(int d, int rep, int B, int R, int W) {
  return (d == 64 || d == 128) && (rep == 1 || rep == 2 || rep % 4 == 0) && rep <= 64 &&
         B <= QR && R <= 16 && W % KC == 0;
}

hipError_t launch_attention_mfma(const AttnArgs& a, int hkv, int batch, hipStream_t st) {
  if (!attention_mfma_supported(a.d, a.rep, a.B, a.R, a.W)) return hipErrorInvalidValue;
  return a.d == 128 ? launch_d<128>(a, hkv, batch, st) : launch_d<64>(a, hkv, batch, st);
}

}  // namespace ldr
