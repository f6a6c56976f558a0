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
// Sum over the block (kThreads threads); every thread gets the result.
__device__ inline float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  __syncthreads();
  if (l == 0) red[w] = v;
  __syncthreads();
  float s = 0.f;
  for (int i = 0; i < kThreads / 64; ++i) s += red[i];
  return s;
}

struct SlotArgs {
  const float* part; long split_stride; int splits;
  const void* embed; const void* mask_emb; const void* pos_emb; const void* fc_norm;
  const void* in_norm0; const int32_t* anchor; const int64_t* pos;
  float* x; void* nrm; float* rope; int32_t* status;
  int hidden, B, d, M, vocab;
  float eps; double base;
};

// One workgroup per (slot i, sequence b): every workgroup of a sequence
// reduces the boundary-fusion partials itself (hidden floats per split, from
// L2) so the slots proceed independently.
template <typename T>
__global__ void __launch_bounds__(kThreads) slot_init_kernel(SlotArgs a) {
  extern __shared__ float smem[];
  float* c = smem;                 // [hidden]
  float* red = smem + a.hidden;    // [4]
  const int i = blockIdx.x, b = blockIdx.y, H = a.hidden;
  const long m = (long)b * a.B + i;
  float ss = 0.f;
  for (int k = threadIdx.x * 4; k < H; k += kThreads * 4) {
    float4 v = *reinterpret_cast<const float4*>(a.part + (long)b * H + k);
    for (int s = 1; s < a.splits; ++s) {
      const float4 u = *reinterpret_cast<const float4*>(a.part + s * a.split_stride + (long)b * H + k);
      v.x += u.x; v.y += u.y; v.z += u.z; v.w += u.w;
    }
    *reinterpret_cast<float4*>(c + k) = v;
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  const float inv_c = rsqrtf(block_sum(ss, red) / H + a.eps);
  int anchor = a.anchor[b];
  if (anchor < 0 || anchor >= a.vocab) {  // never read outside the embedding table
    if (threadIdx.x == 0 && i == 0) atomicOr(a.status, kFlagAnchor);
    anchor = 0;
  }
  const T* e = i == 0 ? static_cast<const T*>(a.embed) + (long)anchor * H
                      : static_cast<const T*>(a.mask_emb);
  const T* p = static_cast<const T*>(a.pos_emb) + (long)i * H;
  const T* gfc = static_cast<const T*>(a.fc_norm);
  float sx = 0.f;
  for (int k = threadIdx.x; k < H; k += kThreads) {
    const float v = Elem<T>::load(e + k) + Elem<T>::load(p + k) +
                    c[k] * inv_c * Elem<T>::load(gfc + k);
    c[k] = v;                      // each thread rewrites only the entries it read
    a.x[m * H + k] = v;
    sx += v * v;
  }
  const float inv = rsqrtf(block_sum(sx, red) / H + a.eps);
  const T* gin = static_cast<const T*>(a.in_norm0);
  for (int k = threadIdx.x; k < H; k += kThreads)
    Elem<T>::store(static_cast<T*>(a.nrm) + m * H + k, c[k] * inv * Elem<T>::load(gin + k));
  // rotary table row of this slot, absolute position t + i
  const int half = a.d / 2;
  const long t = a.pos[b];
  for (int e2 = threadIdx.x; e2 < half; e2 += kThreads) {
    const double inv_freq = pow(a.base, -2.0 * e2 / a.d);
    const double ang = (double)(t + i) * inv_freq;
    a.rope[m * half + e2] = (float)cos(ang);
    a.rope[(long)a.M * half + m * half + e2] = (float)sin(ang);
  }
}

struct ResidArgs {
  const float* part; long split_stride; int splits;
  float* x; void* nrm; const void* gain; int hidden; float eps;
};

template <typename T>
__global__ void __launch_bounds__(kThreads) resid_norm_kernel(ResidArgs a) {
  __shared__ float red[kThreads / 64];
  const long m = blockIdx.x;
  const int H = a.hidden;
  float* x = a.x + m * H;
  const float* part = a.part + m * H;
  float ss = 0.f;
  for (int k = threadIdx.x * 4; k < H; k += kThreads * 4) {
    float4 v = *reinterpret_cast<const float4*>(x + k);
    for (int s = 0; s < a.splits; ++s) {
      const float4 u = *reinterpret_cast<const float4*>(part + s * a.split_stride + k);
      v.x += u.x; v.y += u.y; v.z += u.z; v.w += u.w;
    }
    *reinterpret_cast<float4*>(x + k) = v;
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  const float inv = rsqrtf(block_sum(ss, red) / H + a.eps);
  const T* gain = static_cast<const T*>(a.gain);
  T* out = static_cast<T*>(a.nrm) + m * H;
  for (int k = threadIdx.x * 4; k < H; k += kThreads * 4) {
    const float4 v = *reinterpret_cast<const float4*>(x + k);
    Elem<T>::store(out + k + 0, v.x * inv * Elem<T>::load(gain + k + 0));
    Elem<T>::store(out + k + 1, v.y * inv * Elem<T>::load(gain + k + 1));
    Elem<T>::store(out + k + 2, v.z * inv * Elem<T>::load(gain + k + 2));
    Elem<T>::store(out + k + 3, v.w * inv * Elem<T>::load(gain + k + 3));
  }
}

// Generic attention over the concatenated context, one workgroup per (query
// head h, sequence b): scores for all keys in LDS, one softmax, then P.V.
template <typename T>
__global__ void __launch_bounds__(kThreads) attention_valu_kernel(AttnArgs a) {
  extern __shared__ float smem[];
  const int h = blockIdx.x, b = blockIdx.y, g = h / a.rep;
  const int d = a.d, B = a.B, half = d / 2;
  const long t = a.pos[b];
  const int nv = (int)(t < a.W ? t : a.W);
  const int nsum = t > 0 ? a.R : 0;
  const int NK = B + nv + nsum;
  float* qs = smem;                 // [B][d]
  float* ks = qs + B * d;           // [B][d]
  float* vs = ks + B * d;           // [B][d]
  float* S = vs + B * d;            // [B][B + W + R]
  const int ldS = B + a.W + a.R;

  // q (head h), k and v (group g) of the block, summed over the split-K partials
  for (int idx = threadIdx.x; idx < 3 * B * d; idx += kThreads) {
    const int which = idx / (B * d), i = (idx / d) % B, e = idx % d;
    const int col = which == 0 ? h * d + e
                  : which == 1 ? (a.hq + g) * d + e : (a.hq + a.hkv + g) * d + e;
    const long m = (long)b * B + i;
    float v = 0.f;
    for (int s = 0; s < a.splits; ++s) v += a.part[s * a.split_stride + m * a.qkv_out + col];
    (which == 0 ? qs : which == 1 ? ks : vs)[i * d + e] = v;
  }
  __syncthreads();
  // per-head RMSNorm and rotate-half RoPE on q and k: one wave per row
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int r = wave; r < 2 * B; r += kThreads / 64) {
    float* row = r < B ? qs + r * d : ks + (r - B) * d;
    const T* gain = static_cast<const T*>(r < B ? a.q_norm : a.k_norm);
    const int i = r < B ? r : r - B;
    float ss = 0.f;
    for (int e = lane; e < d; e += 64) ss += row[e] * row[e];
    const float inv = rsqrtf(wave_sum(ss) / d + a.eps);
    const long m = (long)b * B + i;
    for (int e = lane; e < half; e += 64) {
      const float x1 = row[e] * inv * Elem<T>::load(gain + e);
      const float x2 = row[e + half] * inv * Elem<T>::load(gain + e + half);
      const float cs = a.rope[m * half + e], sn = a.rope[(long)a.M * half + m * half + e];
      row[e] = x1 * cs - x2 * sn;
      row[e + half] = x1 * sn + x2 * cs;
    }
  }
  __syncthreads();
  const uint8_t* seq = a.arena + (size_t)b * a.stride;
  const T* Kw = reinterpret_cast<const T*>(seq + a.kw) + ((size_t)(a.layer * a.hkv + g) * a.W) * d;
  const T* Vw = reinterpret_cast<const T*>(seq + a.vw) + ((size_t)(a.layer * a.hkv + g) * a.W) * d;
  const T* Gh = static_cast<const T*>(a.G) + ((size_t)(a.layer * a.hq + h) * a.R) * d;
  const float* Mh = reinterpret_cast<const float*>(seq + a.m_off) + ((size_t)(a.layer * a.hq + h) * a.R) * d;
  for (int idx = threadIdx.x; idx < B * NK; idx += kThreads) {
    const int i = idx / NK, k = idx % NK;
    const float* q = qs + i * d;
    float dot = 0.f;
    if (k < B) {
      for (int e = 0; e < d; ++e) dot += q[e] * ks[k * d + e];
    } else if (k < B + nv) {
      const T* kr = Kw + (size_t)(k - B) * d;
      for (int e = 0; e < d; ++e) dot += q[e] * Elem<T>::load(kr + e);
    } else {
      const T* kr = Gh + (size_t)(k - B - nv) * d;
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
    for (int k = 0; k < nv; ++k) acc += p[B + k] * Elem<T>::load(Vw + (size_t)k * d + e);
    for (int k = 0; k < nsum; ++k) acc += p[B + nv + k] * Mh[(size_t)k * d + e];
    Elem<T>::store(out + ((long)b * B + i) * (a.hq * d) + h * d + e, acc);
  }
}

}  // namespace

hipError_t launch_slot_init(const Shape& s, int batch, const DraftPtrs& p, int fc_splits,
                            const ldr_weights* w, const int32_t* anchor, hipStream_t st) {
  SlotArgs a;
  a.part = p.part; a.split_stride = (long)batch * s.hidden; a.splits = fc_splits;
  a.embed = w->embed; a.mask_emb = w->mask_emb; a.pos_emb = w->pos_emb; a.fc_norm = w->fc_norm;
  a.in_norm0 = w->layers[0].in_norm; a.anchor = anchor; a.pos = p.pos;
  a.x = p.x; a.nrm = p.nrm; a.rope = p.rope; a.status = p.status;
  a.hidden = s.hidden; a.B = s.B; a.d = s.d; a.M = batch * s.B; a.vocab = s.vocab;
  a.eps = s.eps; a.base = s.rope_base;
  const size_t shm = (s.hidden + 4) * sizeof(float);
  if (s.dtype == LDR_BF16)
    hipLaunchKernelGGL(slot_init_kernel<uint16_t>, dim3(s.B, batch), dim3(kThreads), shm, st, a);
  else
    hipLaunchKernelGGL(slot_init_kernel<float>, dim3(s.B, batch), dim3(kThreads), shm, st, a);
  return hipGetLastError();
}

hipError_t launch_resid_norm(const Shape& s, int M, const DraftPtrs& p, int splits,
                             const void* gain, hipStream_t st) {
  ResidArgs a;
  a.part = p.part; a.split_stride = (long)M * s.hidden; a.splits = splits;
  a.x = p.x; a.nrm = p.nrm; a.gain = gain; a.hidden = s.hidden; a.eps = s.eps;
  if (s.dtype == LDR_BF16)
    hipLaunchKernelGGL(resid_norm_kernel<uint16_t>, dim3(M), dim3(kThreads), 0, st, a);
  else
    hipLaunchKernelGGL(resid_norm_kernel<float>, dim3(M), dim3(kThreads), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_attention(const Shape& s, const Layout& L, int batch, const DraftPtrs& p,
                            int qkv_splits, int layer, const ldr_layer_weights* lw,
                            hipStream_t st) {
  AttnArgs a;
  const int M = batch * s.B;
  a.part = p.part; a.split_stride = (long)M * s.qkv_out; a.splits = qkv_splits;
  a.arena = p.arena; a.stride = L.stride; a.kw = L.kw; a.vw = L.vw; a.m_off = L.m;
  a.pos = p.pos; a.G = p.G; a.rope = p.rope; a.q_norm = lw->q_norm; a.k_norm = lw->k_norm;
  a.o = p.o; a.layer = layer; a.hq = s.hq; a.hkv = s.hkv; a.d = s.d; a.B = s.B; a.W = s.W;
  a.R = s.R; a.rep = s.rep; a.qkv_out = s.qkv_out; a.M = M;
  a.eps = s.eps; a.inv_sqrt_d = 1.0f / sqrtf((float)s.d);
  const size_t shm = (size_t)(3 * s.B * s.d + s.B * (s.B + s.W + s.R)) * sizeof(float);
  if (s.dtype == LDR_BF16) return launch_attention_mfma(a, s.hkv, batch, st);
  const dim3 grid(s.hq, batch);
  hipLaunchKernelGGL(attention_valu_kernel<float>, grid, dim3(kThreads), shm, st, a);
  return hipGetLastError();
}

}  // namespace ldr
