// Draft-step kernels around the GEMMs (Sec. 2.3; Eq. 6; App. A.1):
//  * slot_init: sums the boundary-fusion split-K partials, c = RMSNorm(.),
//    x_i = E[u_i] + P_i + c, the first layer's pre-norm, and the per-slot
//    rotary cos/sin table (angles pos * base^(-2e/d) in double, rounded to
//    fp32 once);
//  * resid_norm: x += sum of split-K partials, then RMSNorm(x) for the next
//    GEMM;
//  * attention: per (query head, sequence), q/k RMSNorm + RoPE on the block's
//    own q and k, then one softmax over [block; window; summary] keys.
#include "ldr_internal.h"

namespace ldr {
namespace {

constexpr int kThreads = 256;

__device__ inline float wave_sum(float v) {
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
  return v;
}
__device__ inline float wave_max(float v) {
  for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off));
  return v;
}
// Sum over the block (NT threads); every thread gets the result.
template <int NT = kThreads>
__device__ inline float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  __syncthreads();
  if (l == 0) red[w] = v;
  __syncthreads();
  float s = 0.f;
  for (int i = 0; i < NT / 64; ++i) s += red[i];
  return s;
}

struct SlotArgs {
  const float* part; long split_stride; int splits;
  int use_c;   // 0: no boundary view (ablation variant), c = 0
  const void* embed; const void* mask_emb; const void* pos_emb; const void* fc_norm;
  const void* in_norm0; const int32_t* anchor; const int64_t* pos;
  float* x; void* nrm; float* rope; int32_t* status;
  int frag;   // nrm in the fragment layout (else row-major)
  int hidden, B, d, M, vocab;
  float eps; double base;
};

// Loads and stores of 4 consecutive elements of the configuration dtype.
template <typename T> struct Vec4;
template <> struct Vec4<float> {
  __device__ static float4 load(const float* p) { return *reinterpret_cast<const float4*>(p); }
  __device__ static void store(float* p, float4 v) { *reinterpret_cast<float4*>(p) = v; }
};
template <> struct Vec4<uint16_t> {
  __device__ static float4 load(const uint16_t* p) {
    const uint2 u = *reinterpret_cast<const uint2*>(p);
    return make_float4(bf16_to_f32(u.x & 0xffffu), bf16_to_f32(u.x >> 16),
                       bf16_to_f32(u.y & 0xffffu), bf16_to_f32(u.y >> 16));
  }
  __device__ static void store(uint16_t* p, float4 v) {
    uint2 u;
    u.x = f32_to_bf16(v.x) | ((uint32_t)f32_to_bf16(v.y) << 16);
    u.y = f32_to_bf16(v.z) | ((uint32_t)f32_to_bf16(v.w) << 16);
    *reinterpret_cast<uint2*>(p) = u;
  }
};
__device__ inline float4 f4add(float4 a, float4 b) {
  return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w);
}
__device__ inline float f4dot(float4 a) { return a.x * a.x + a.y * a.y + a.z * a.z + a.w * a.w; }
__device__ inline float4 f4scale(float4 a, float s, float4 g) {
  return make_float4(a.x * s * g.x, a.y * s * g.y, a.z * s * g.z, a.w * s * g.w);
}

// The row kernels below (slot init, residual norm) take one workgroup of
// kNormThreads threads per row of `hidden` <= kMaxHidden elements: each
// thread owns float4 chunk c of (threadIdx + c * kNormThreads) for
// c < kNormChunks, so a row of up to 4096 elements is one float4 per thread,
// and every CU keeps 16 waves of loads in flight. The loops over chunks and
// splits have compile-time bounds, so every load is issued before the first
// reduction instead of one memory round trip per loop iteration.
constexpr int kMaxHidden = 8192;
constexpr int kNormThreads = 1024, kNormChunks = kMaxHidden / (kNormThreads * 4);

// One workgroup per (slot i, sequence b); every workgroup of a sequence
// reduces the boundary-fusion partials itself (from L2).
template <typename T, int SPLITS>
__global__ void __launch_bounds__(kNormThreads) slot_init_kernel(SlotArgs a) {
  __shared__ float red[kNormThreads / 64];
  const int H = a.hidden;
  const int i = blockIdx.x, b = blockIdx.y;
  const long m = (long)b * a.B + i;
  int anchor = a.anchor[b];
  if (anchor < 0 || anchor >= a.vocab) {  // never read outside the embedding table
    if (threadIdx.x == 0 && i == 0) atomicOr(a.status, kFlagAnchor);
    anchor = 0;
  }
  const T* e = i == 0 ? static_cast<const T*>(a.embed) + (long)anchor * H
                      : static_cast<const T*>(a.mask_emb);
  const T* p = static_cast<const T*>(a.pos_emb) + (long)i * H;
  // rotary table row of this slot, absolute position t + i (fp64 pow, cos
  // and sin, before the row's loads: at the end of the kernel they took
  // 1.5 us more)
  const int half = a.d / 2;
  const long t = a.pos[b];
  for (int e2 = threadIdx.x; e2 < half; e2 += kNormThreads) {
    const double inv_freq = pow(a.base, -2.0 * e2 / a.d);
    const double ang = (double)(t + i) * inv_freq;
    a.rope[m * half + e2] = (float)cos(ang);
    a.rope[(long)a.M * half + m * half + e2] = (float)sin(ang);
  }
  float4 c[kNormChunks], ep[kNormChunks], gfc[kNormChunks], gin[kNormChunks];
  float ss = 0.f;
#pragma unroll
  for (int ch = 0; ch < kNormChunks; ++ch) {
    const int k = (threadIdx.x + ch * kNormThreads) * 4;
    if (k < H) {
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
      gfc[ch] = v;
      if (a.use_c) {
        v = *reinterpret_cast<const float4*>(a.part + (long)b * H + k);
#pragma unroll
        for (int s = 1; s < SPLITS; ++s)
          v = f4add(v, *reinterpret_cast<const float4*>(a.part + s * a.split_stride + (long)b * H + k));
        gfc[ch] = Vec4<T>::load(static_cast<const T*>(a.fc_norm) + k);
      }
      c[ch] = v;
      ep[ch] = f4add(Vec4<T>::load(e + k), Vec4<T>::load(p + k));
      gin[ch] = Vec4<T>::load(static_cast<const T*>(a.in_norm0) + k);
      ss += f4dot(v);
    }
  }
  const float inv_c = rsqrtf(block_sum<kNormThreads>(ss, red) / H + a.eps);
  float sx = 0.f;
#pragma unroll
  for (int ch = 0; ch < kNormChunks; ++ch) {
    const int k = (threadIdx.x + ch * kNormThreads) * 4;
    if (k < H) {
      c[ch] = f4add(ep[ch], f4scale(c[ch], inv_c, gfc[ch]));
      *reinterpret_cast<float4*>(a.x + m * H + k) = c[ch];
      sx += f4dot(c[ch]);
    }
  }
  const float inv = rsqrtf(block_sum<kNormThreads>(sx, red) / H + a.eps);
#pragma unroll
  for (int ch = 0; ch < kNormChunks; ++ch) {
    const int k = (threadIdx.x + ch * kNormThreads) * 4;
    if (k < H) {
      // four consecutive k stay inside one 16-byte chunk of the fragment layout
      const long o = a.frag ? ((m >> 4) * (long)(H >> 5) + (k >> 5)) * 512 +
                                  ((k >> 3) & 3) * 128 + (m & 15) * 8 + (k & 7)
                            : m * H + k;
      Vec4<T>::store(static_cast<T*>(a.nrm) + o, f4scale(c[ch], inv, gin[ch]));
    }
  }
}

struct ResidArgs {
  const float* part; long split_stride; int splits;
  float* x; void* nrm; const void* gain; int hidden; float eps;
  int layout;  // nrm layout: NRM_ROWS, NRM_TILED or NRM_FRAG (hidden % 32 == 0)
};

template <typename T, int SPLITS>
__global__ void __launch_bounds__(kNormThreads) resid_norm_kernel(ResidArgs a) {
  __shared__ float red[kNormThreads / 64];
  const long m = blockIdx.x;
  const int H = a.hidden;
  float* x = a.x + m * H;
  const float* part = a.part + m * H;
  float4 v[kNormChunks], g[kNormChunks];
  float ss = 0.f;
#pragma unroll
  for (int ch = 0; ch < kNormChunks; ++ch) {
    const int k = (threadIdx.x + ch * kNormThreads) * 4;
    if (k < H) {
      float4 u = *reinterpret_cast<const float4*>(x + k);
#pragma unroll
      for (int s = 0; s < SPLITS; ++s)
        u = f4add(u, *reinterpret_cast<const float4*>(part + s * a.split_stride + k));
      v[ch] = u;
      g[ch] = Vec4<T>::load(static_cast<const T*>(a.gain) + k);
      ss += f4dot(u);
    }
  }
  const float inv = rsqrtf(block_sum<kNormThreads>(ss, red) / H + a.eps);
  T* out = static_cast<T*>(a.nrm);
  const long rbase = a.layout == NRM_TILED ? (m >> 8) * (long)(H >> 5) * 8192 + (m & 255) * 32
                   : a.layout == NRM_FRAG ? (m >> 4) * (long)(H >> 5) * 512 + (m & 15) * 8
                                          : m * H;
#pragma unroll
  for (int ch = 0; ch < kNormChunks; ++ch) {
    const int k = (threadIdx.x + ch * kNormThreads) * 4;
    if (k < H) {
      *reinterpret_cast<float4*>(x + k) = v[ch];
      // four consecutive k stay inside one 16-byte chunk of either tiled layout
      const long o = a.layout == NRM_TILED ? rbase + (long)(k >> 5) * 8192 + (k & 31)
                   : a.layout == NRM_FRAG ? rbase + (long)(k >> 5) * 512 + ((k >> 3) & 3) * 128 +
                                                (k & 7)
                                          : rbase + k;
      Vec4<T>::store(out + o, f4scale(v[ch], inv, g[ch]));
    }
  }
}

struct QkvArgs {
  const float* part; long split_stride;   // QKV split-K partials [splits][M][qkv_out]
  void* out;                              // [M][qkv_out] of the configuration dtype
  const void* q_norm; const void* k_norm; // per-head RMSNorm gains [d]
  const float* rope;                      // cos / sin [M][d/2] each
  int M, nh, hq, hkv, d, qkv_out;
  float eps;
};

// Block q, k and v rows (Eq. 6 inputs) for fp32 models (the bf16 attention
// kernel does this in its prologue): sum of the split-K partials, then for
// q and k heads the per-head RMSNorm and the rotate-half RoPE at position
// t + i (table of slot_init). One wave per (row m, head slot hs), where slots
// [0, hq) are query heads, [hq, hq + hkv) key heads and the rest value heads;
// lane e < d/2 owns the rotary pair (e, e + d/2).
template <typename T, int SPLITS>
__global__ void __launch_bounds__(kThreads) qkv_finish_kernel(QkvArgs a) {
  const long wid = (long)blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
  if (wid >= (long)a.M * a.nh) return;  // whole waves only
  const int lane = threadIdx.x & 63, half = a.d / 2;
  const long m = wid / a.nh;
  const int hs = (int)(wid % a.nh);
  const float* src = a.part + m * a.qkv_out + (long)hs * a.d;
  float x1 = 0.f, x2 = 0.f;
  if (lane < half) {
    float p1[SPLITS], p2[SPLITS];
#pragma unroll
    for (int s = 0; s < SPLITS; ++s) {
      p1[s] = src[s * a.split_stride + lane];
      p2[s] = src[s * a.split_stride + lane + half];
    }
#pragma unroll
    for (int s = 0; s < SPLITS; ++s) { x1 += p1[s]; x2 += p2[s]; }
  }
  if (hs < a.hq + a.hkv) {
    const float inv = rsqrtf(wave_sum(x1 * x1 + x2 * x2) / a.d + a.eps);
    if (lane < half) {
      const T* gain = static_cast<const T*>(hs < a.hq ? a.q_norm : a.k_norm);
      const float z1 = x1 * inv * Elem<T>::load(gain + lane);
      const float z2 = x2 * inv * Elem<T>::load(gain + lane + half);
      const float cs = a.rope[m * half + lane];
      const float sn = a.rope[(long)a.M * half + m * half + lane];
      x1 = z1 * cs - z2 * sn;
      x2 = z1 * sn + z2 * cs;
    }
  }
  if (lane < half) {
    T* dst = static_cast<T*>(a.out) + m * a.qkv_out + (long)hs * a.d;
    Elem<T>::store(dst + lane, x1);
    Elem<T>::store(dst + lane + half, x2);
  }
}

// Generic attention over the concatenated context, one workgroup per (query
// head h, sequence b): scores for all keys in LDS, one softmax, then P.V.
template <typename T>
__global__ void __launch_bounds__(kThreads) attention_valu_kernel(AttnArgs a) {
  extern __shared__ float smem[];
  const int h = blockIdx.x, b = blockIdx.y, g = h / a.rep;
  const int d = a.d, B = a.B;
  const long t = a.pos[b];
  // keys: block, valid window rows, the valid slots of the two pooled banks
  // (mean-pooled summary; slot k valid once k chunks have begun), the learned
  // summary entries
  const int nv = (int)(t < a.W ? t : a.W);
  const int np0 = a.P ? (int)min((t + a.S0 - 1) / a.S0, (long)a.P) : 0;
  const int np1 = a.P ? (int)min((t + a.S1 - 1) / a.S1, (long)a.P) : 0;
  const int nsum = t > 0 && a.use_summary ? a.R : 0;
  const int NK = B + nv + np0 + np1 + nsum;
  float* qs = smem;                 // [B][d]
  float* ks = qs + B * d;           // [B][d]
  float* vs = ks + B * d;           // [B][d]
  float* S = vs + B * d;            // [B][B + W + R]
  const int ldS = B + a.Wx + a.R;

  // q (head h), k and v (group g) of the block
  const T* qkv = static_cast<const T*>(a.qkv);
  for (int idx = threadIdx.x; idx < 3 * B * d; idx += kThreads) {
    const int which = idx / (B * d), i = (idx / d) % B, e = idx % d;
    const int col = which == 0 ? h * d + e
                  : which == 1 ? (a.hq + g) * d + e : (a.hq + a.hkv + g) * d + e;
    (which == 0 ? qs : which == 1 ? ks : vs)[i * d + e] =
        Elem<T>::load(qkv + ((long)b * B + i) * a.qkv_out + col);
  }
  __syncthreads();
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const uint8_t* seq = a.arena + (size_t)b * a.stride;
  const T* Kw = reinterpret_cast<const T*>(seq + a.kw) + ((size_t)(a.layer * a.hkv + g) * a.Wx) * d;
  const T* Vw = reinterpret_cast<const T*>(seq + a.vw) + ((size_t)(a.layer * a.hkv + g) * a.Wx) * d;
  // region row of key k - B among the window and pooled keys
  auto region_row = [&](int k) -> int {
    return k < nv ? k : k < nv + np0 ? a.W + (k - nv) : a.W + a.P + (k - nv - np0);
  };
  const int nreg = nv + np0 + np1;
  const T* Gh = nsum ? static_cast<const T*>(a.G) + ((size_t)(a.layer * a.hq + h) * a.R) * d
                     : nullptr;
  const float* Mh = reinterpret_cast<const float*>(seq + a.m_off) + ((size_t)(a.layer * a.hq + h) * a.R) * d;
  for (int idx = threadIdx.x; idx < B * NK; idx += kThreads) {
    const int i = idx / NK, k = idx % NK;
    const float* q = qs + i * d;
    float dot = 0.f;
    if (k < B) {
      for (int e = 0; e < d; ++e) dot += q[e] * ks[k * d + e];
    } else if (k < B + nreg) {
      const T* kr = Kw + (size_t)region_row(k - B) * d;
      for (int e = 0; e < d; ++e) dot += q[e] * Elem<T>::load(kr + e);
    } else {
      const T* kr = Gh + (size_t)(k - B - nreg) * d;
      for (int e = 0; e < d; ++e) dot += q[e] * Elem<T>::load(kr + e);
    }
    S[i * ldS + k] = dot * a.inv_sqrt_d;
  }
  __syncthreads();
  for (int i = wave; i < B; i += kThreads / 64) {
    float mx = -INFINITY;
    for (int k = lane; k < NK; k += 64) mx = fmaxf(mx, S[i * ldS + k]);
    mx = wave_max(mx);
    float sum = 0.f;
    for (int k = lane; k < NK; k += 64) {
      const float p = expf(S[i * ldS + k] - mx);
      S[i * ldS + k] = p;
      sum += p;
    }
    const float inv = 1.f / wave_sum(sum);
    for (int k = lane; k < NK; k += 64) S[i * ldS + k] *= inv;
  }
  __syncthreads();
  T* out = static_cast<T*>(a.o);
  for (int idx = threadIdx.x; idx < B * d; idx += kThreads) {
    const int i = idx / d, e = idx % d;
    const float* p = S + i * ldS;
    float acc = 0.f;
    for (int k = 0; k < B; ++k) acc += p[k] * vs[k * d + e];
    for (int k = 0; k < nreg; ++k)
      acc += p[B + k] * Elem<T>::load(Vw + (size_t)e * a.Wx + region_row(k));
    for (int k = 0; k < nsum; ++k) acc += p[B + nreg + k] * Mh[(size_t)k * d + e];
    Elem<T>::store(out + ((long)b * B + i) * (a.hq * d) + h * d + e, acc);
  }
}

struct SlotLaunch {
  template <typename T, int S>
  static void go(dim3 grid, const SlotArgs& a, hipStream_t st) {
    hipLaunchKernelGGL((slot_init_kernel<T, S>), grid, dim3(kNormThreads), 0, st, a);
  }
};
struct QkvLaunch {
  template <typename T, int S>
  static void go(dim3 grid, const QkvArgs& a, hipStream_t st) {
    hipLaunchKernelGGL((qkv_finish_kernel<T, S>), grid, dim3(kThreads), 0, st, a);
  }
};
struct ResidLaunch {
  template <typename T, int S>
  static void go(dim3 grid, const ResidArgs& a, hipStream_t st) {
    hipLaunchKernelGGL((resid_norm_kernel<T, S>), grid, dim3(kNormThreads), 0, st, a);
  }
};
// Dispatch on the split-K factor (1, 2, 4 or 8).
template <typename T, typename L, typename Args>
hipError_t launch_split(int splits, dim3 grid, const Args& a, hipStream_t st) {
  switch (splits) {
    case 1: L::template go<T, 1>(grid, a, st); break;
    case 2: L::template go<T, 2>(grid, a, st); break;
    case 4: L::template go<T, 4>(grid, a, st); break;
    case 8: L::template go<T, 8>(grid, a, st); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

bool norm_hidden_supported(int hidden) { return hidden % 4 == 0 && hidden <= kMaxHidden; }

hipError_t launch_slot_init(const Shape& s, int batch, const DraftPtrs& p, int fc_splits,
                            const ldr_weights* w, const int32_t* anchor, hipStream_t st,
                            void* frag_out) {
  SlotArgs a;
  a.part = p.part; a.split_stride = (long)batch * s.hidden; a.splits = fc_splits;
  a.use_c = s.keep_bnd;
  a.embed = w->embed; a.mask_emb = w->mask_emb; a.pos_emb = w->pos_emb; a.fc_norm = w->fc_norm;
  a.in_norm0 = w->layers[0].in_norm; a.anchor = anchor; a.pos = p.pos;
  a.x = p.x; a.nrm = frag_out ? frag_out : p.nrm; a.rope = p.rope; a.status = p.status;
  a.frag = frag_out != nullptr;
  a.hidden = s.hidden; a.B = s.B; a.d = s.d; a.M = batch * s.B; a.vocab = s.vocab;
  a.eps = s.eps; a.base = s.rope_base;
  return s.dtype == LDR_BF16 ? launch_split<uint16_t, SlotLaunch>(fc_splits, dim3(s.B, batch), a, st)
                            : launch_split<float, SlotLaunch>(fc_splits, dim3(s.B, batch), a, st);
}

hipError_t launch_resid_norm(const Shape& s, int M, const DraftPtrs& p, int splits,
                             const void* gain, hipStream_t st, void* tiled_out, int layout) {
  ResidArgs a;
  a.part = p.part; a.split_stride = (long)M * s.hidden; a.splits = splits;
  a.x = p.x; a.nrm = tiled_out ? tiled_out : p.nrm; a.gain = gain; a.hidden = s.hidden;
  a.eps = s.eps; a.layout = tiled_out ? layout : NRM_ROWS;
  return s.dtype == LDR_BF16 ? launch_split<uint16_t, ResidLaunch>(splits, dim3(M), a, st)
                            : launch_split<float, ResidLaunch>(splits, dim3(M), a, st);
}

hipError_t launch_qkv_finish(const Shape& s, int M, const DraftPtrs& p, int splits,
                             const ldr_layer_weights* lw, hipStream_t st) {
  QkvArgs a;
  a.part = p.part; a.split_stride = (long)M * s.qkv_out; a.out = p.qkv;
  a.q_norm = lw->q_norm; a.k_norm = lw->k_norm; a.rope = p.rope;
  a.M = M; a.nh = s.hq + 2 * s.hkv; a.hq = s.hq; a.hkv = s.hkv; a.d = s.d;
  a.qkv_out = s.qkv_out; a.eps = s.eps;
  const int waves = kThreads / 64;
  const dim3 grid((unsigned)(((long)M * a.nh + waves - 1) / waves));
  if (s.dtype == LDR_BF16) return hipErrorInvalidValue;   // the bf16 attention finishes q/k/v
  return launch_split<float, QkvLaunch>(splits, grid, a, st);
}

hipError_t launch_attention(const Shape& s, const Layout& L, int batch, const DraftPtrs& p,
                            int layer, const ldr_layer_weights* lw, int qkv_splits,
                            hipStream_t st, bool o_frag) {
  AttnArgs a;
  a.qkv = p.qkv;
  a.part = p.part; a.split_stride = (long)batch * s.B * s.qkv_out; a.splits = qkv_splits;
  a.rows = batch * s.B; a.q_norm = lw->q_norm; a.k_norm = lw->k_norm; a.rope = p.rope;
  a.eps = s.eps;
  a.arena = p.arena; a.stride = L.stride; a.kw = L.kw; a.vw = L.vw; a.m_off = L.m;
  a.pos = p.pos; a.G = p.G;
  a.o = p.o; a.layer = layer; a.hq = s.hq; a.hkv = s.hkv; a.d = s.d; a.B = s.B; a.W = s.Wr;
  a.Wx = s.Wx; a.P = s.P; a.S0 = s.S0; a.S1 = s.S1;
  a.R = s.R; a.rep = s.rep; a.qkv_out = s.qkv_out;
  a.use_summary = s.learned;
  a.inv_sqrt_d = 1.0f / sqrtf((float)s.d);
  a.o_frag = o_frag && s.dtype == LDR_BF16;
  const size_t shm = (size_t)(3 * s.B * s.d + s.B * (s.B + s.Wx + s.R)) * sizeof(float);
  if (s.dtype == LDR_BF16) return launch_attention_mfma(a, s.hkv, batch, st);
  const dim3 grid(s.hq, batch);
  hipLaunchKernelGGL(attention_valu_kernel<float>, grid, dim3(kThreads), shm, st, a);
  return hipGetLastError();
}

}  // namespace ldr
