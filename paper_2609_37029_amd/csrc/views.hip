// Fixed-size context views on the GPU (Sec. 2.2; App. A.2, Eq. 10-11).
//
// One workgroup per (kv group g, layer j, sequence b) ingests the new rows of
// that sequence for that head group, reading each new row once:
//  * ring write of the last min(n, W) rows into window slots (t + r) mod W;
//    K rows as they come ([W][d]), V transposed ([d][W]) so that attention
//    reads V with the key index contiguous, as its P.V contraction needs;
//  * for the rep * R summary queries of the group's query heads, the
//    statistics of the new set N (Eq. 10) by a tiled online log-sum-exp over
//    the rows, then the two-way merge with the stored (eta, m) (Eq. 11);
//  * a slice of the boundary-state copy.
// The commit then advances t (or raises the sticky range flag): the last
// workgroup of the last kernel that reads t does it, once every other
// workgroup of that launch has counted itself done on a device counter (each
// counts after its own reads of t), so every workgroup reads the old t and
// no separate launch is needed; without new rows a one-thread-per-sequence
// commit kernel does it.
#include "ldr_internal.h"

namespace ldr {
namespace {

constexpr int kThreads = 256;
constexpr int kTileRows = 32;   // rows of N staged in LDS per step

__global__ void __launch_bounds__(kThreads)
views_reset_kernel(uint8_t* arena, size_t stride, size_t eta_off, size_t eta_bytes,
                   int batch, int64_t* pos) {
  const size_t words = stride / 4;
  const size_t total = words * (size_t)batch;
  uint32_t* w = reinterpret_cast<uint32_t*>(arena);
  for (size_t i = blockIdx.x * (size_t)kThreads + threadIdx.x; i < total;
       i += (size_t)gridDim.x * kThreads) {
    const size_t off = (i % words) * 4;
    const bool is_eta = off >= eta_off && off < eta_off + eta_bytes;
    w[i] = is_eta ? 0xff800000u : 0u;  // -inf log-normalizer, zero elsewhere
  }
  if (blockIdx.x == 0)
    for (int b = threadIdx.x; b < batch; b += kThreads) pos[b] = 0;
}

// The commit by the last workgroup of a launch (done == null: not this launch).
struct CommitTail {
  int32_t* done;      // device counter, 0 between launches
  int total;          // workgroups of the launch
  int64_t* pos; const int32_t* n_new; int max_new, batch; int32_t* status;
};

__device__ void commit_tail(const CommitTail& c) {
  if (!c.done) return;
  __shared__ int last;
  __syncthreads();   // every thread of the workgroup is past its reads of t
  if (threadIdx.x == 0) last = atomicAdd(c.done, 1) == c.total - 1;
  __syncthreads();
  if (!last) return;
  for (int b = (int)threadIdx.x; b < c.batch; b += (int)blockDim.x) {
    const int n = c.n_new[b];
    if (n < 0 || n > c.max_new)
      atomicOr(c.status, kFlagRange);
    else
      c.pos[b] += n;
  }
  if (threadIdx.x == 0) atomicExch(c.done, 0);   // ready for the next launch
}

struct UpdateArgs {
  uint8_t* arena; size_t stride; size_t kw, vw, m, eta, h;
  const int64_t* pos; const void* G; const int32_t* n_new; int max_new;
  const void* K_new; const void* V_new; const void* h_new;
  int D, hq, hkv, d, W, R, rep, hb_elems;  // hb_elems = L_b * hidden
  int keep_win, keep_sum, keep_bnd;         // views kept (ablation variants drop some)
  int Wx;                                   // rows per (layer, group) region (window first)
  float inv_sqrt_d;
  CommitTail ct;
};

// Sum over aligned groups of tpq lanes (tpq a power of two): DPP lane swaps
// inside rows of 16 (after each step every lane of a group holds the same
// value), cross-row shuffles beyond.
__device__ inline float group_sum(float v, int tpq) {
  if (tpq >= 2) v += dpp<0xB1>(v);
  if (tpq >= 4) v += dpp<0x4E>(v);
  if (tpq >= 8) v += dpp<0x141>(v);
  if (tpq >= 16) v += dpp<0x140>(v);
  for (int off = 16; off < tpq; off <<= 1) v += __shfl_xor(v, off);
  return v;
}

// 16-byte copy of `n16` chunks.
__device__ inline void copy16(void* dst, const void* src, int idx) {
  reinterpret_cast<uint4*>(dst)[idx] = reinterpret_cast<const uint4*>(src)[idx];
}

// This workgroup's slice of the boundary-state copy (the D * H_kv workgroups
// of a sequence share it).
template <typename T>
__device__ inline void boundary_slice(const UpdateArgs& a, uint8_t* seq, int j, int g, int b,
                                      int nthreads) {
  const int chunks = a.hb_elems * (int)sizeof(T) / 16;
  const int wgs = a.D * a.hkv, wid = j * a.hkv + g;
  const int per = (chunks + wgs - 1) / wgs;
  const int c0 = wid * per, c1 = min(chunks, c0 + per);
  T* hdst = reinterpret_cast<T*>(seq + a.h);
  const T* hsrc = reinterpret_cast<const T*>(a.h_new) + (size_t)b * a.hb_elems;
  for (int c = c0 + (int)threadIdx.x; c < c1; c += nthreads) copy16(hdst, hsrc, c);
}

// DPT: dims of the head each thread owns; TPQ = d / DPT threads share one
// summary query, Q = rep * R queries per workgroup, Q * TPQ = kThreads.
template <typename T, int DPT>
__device__ __forceinline__ void views_update_body(const UpdateArgs& a) {
  const int g = blockIdx.x, j = blockIdx.y, b = blockIdx.z;
  const int n = a.n_new[b];
  if (n <= 0 || n > a.max_new) return;  // empty set: identity; bad count: commit flags it
  const int64_t t = a.pos[b];
  const int d = a.d;
  uint8_t* seq = a.arena + (size_t)b * a.stride;

  // Summary query q of the group is (head g*rep + q / R, summary row q % R);
  // the group's queries are contiguous in G, M and eta. TPQ = d / DPT threads
  // share a query; thread `part` owns dims (c * TPQ + part) * 4 + e.
  constexpr int NV = DPT / 4;         // float4 chunks per thread
  const int tpq = d / DPT;
  const int q = threadIdx.x / tpq;
  const int part = threadIdx.x % tpq;
  const size_t qrow = ((size_t)j * a.hq + g * a.rep) * a.R + q;
  float* Mq = reinterpret_cast<float*>(seq + a.m) + qrow * d;
  float* etaq = reinterpret_cast<float*>(seq + a.eta) + qrow;

  // The stored (eta, m) and the query are loaded first: the stores below go
  // to the same arena, so these loads could not be moved ahead of them.
  const bool sum = a.keep_sum, win = a.keep_win;
  const float eta_a = sum ? *etaq : -INFINITY;
  float4 ma[NV];
  float gq[DPT], acc[DPT];
#pragma unroll
  for (int i = 0; i < DPT; ++i) gq[i] = acc[i] = 0.f;
#pragma unroll
  for (int c = 0; c < NV; ++c) ma[c] = make_float4(0.f, 0.f, 0.f, 0.f);
  if (sum) {
    const T* Gp = reinterpret_cast<const T*>(a.G) + qrow * d;
#pragma unroll
    for (int c = 0; c < NV; ++c) {
      const int dim = (c * tpq + part) * 4;
      ma[c] = *reinterpret_cast<const float4*>(Mq + dim);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        gq[c * 4 + e] = Elem<T>::load(Gp + dim + e) * a.inv_sqrt_d;
        acc[c * 4 + e] = 0.f;
      }
    }
  }

  if (a.keep_bnd) boundary_slice<T>(a, seq, j, g, b, kThreads);

  // ---- rows of the new set N, tile by tile: window ring write of the last
  // min(n, W) rows (slot (t + r) mod W) and the tiled online log-sum-exp ----
  __shared__ float Ks[kTileRows][256 + 4];
  __shared__ float Vs[kTileRows][256 + 4];
  constexpr int EPC = 16 / sizeof(T);  // elements per 16-byte chunk
  T* Kw = reinterpret_cast<T*>(seq + a.kw) + ((size_t)(j * a.hkv + g) * a.Wx) * d;
  T* Vw = reinterpret_cast<T*>(seq + a.vw) + ((size_t)(j * a.hkv + g) * a.Wx) * d;
  float mx = -INFINITY, l = 0.f;
  for (int r0 = 0; r0 < ((win || sum) ? n : 0); r0 += kTileRows) {
    const int nr = min(kTileRows, n - r0);
    __syncthreads();
    const int cpr = d / EPC;
    for (int i = threadIdx.x; i < nr * cpr; i += kThreads) {
      const int r = i / cpr, e0 = (i % cpr) * EPC;
      const size_t src = ((((size_t)b * a.max_new + r0 + r) * a.D + j) * a.hkv + g) * d + e0;
      const uint4 kv = *reinterpret_cast<const uint4*>(reinterpret_cast<const T*>(a.K_new) + src);
      const uint4 vv = *reinterpret_cast<const uint4*>(reinterpret_cast<const T*>(a.V_new) + src);
      if (win && r0 + r >= n - a.W) {  // only the last W rows can survive in the ring
        const size_t slot = (size_t)((t + r0 + r) % a.W);
        *reinterpret_cast<uint4*>(Kw + slot * d + e0) = kv;
      }
      const T* kp = reinterpret_cast<const T*>(&kv);
      const T* vp = reinterpret_cast<const T*>(&vv);
#pragma unroll
      for (int e = 0; e < EPC; ++e) {
        Ks[r][e0 + e] = Elem<T>::load(kp + e);
        Vs[r][e0 + e] = Elem<T>::load(vp + e);
      }
    }
    __syncthreads();
    {  // window V, transposed: lanes take consecutive rows of one dim, whose
       // slots are contiguous (apart from the wrap of the ring)
      const int rs = max(0, n - a.W - r0);  // first row of the tile that survives
      const int r = threadIdx.x % kTileRows;
      if (win && r >= rs && r < nr) {
        const size_t slot = (size_t)((t + r0 + r) % a.W);
        for (int e = threadIdx.x / kTileRows; e < d; e += kThreads / kTileRows)
          Elem<T>::store(Vw + (size_t)e * a.Wx + slot, Vs[r][e]);
      }
    }
    if (!sum) continue;   // window only: no statistics
    float s[kTileRows];
    float tmax = -INFINITY;
#pragma unroll
    for (int r = 0; r < kTileRows; ++r) {
      float p = 0.f;
      if (r < nr) {
#pragma unroll
        for (int c = 0; c < NV; ++c) {
          const float4 k4 = *reinterpret_cast<const float4*>(&Ks[r][(c * tpq + part) * 4]);
          p += gq[c * 4 + 0] * k4.x + gq[c * 4 + 1] * k4.y + gq[c * 4 + 2] * k4.z +
               gq[c * 4 + 3] * k4.w;
        }
      }
      p = group_sum(p, tpq);
      s[r] = r < nr ? p : -INFINITY;
      tmax = fmaxf(tmax, s[r]);
    }
    const float nm = fmaxf(mx, tmax);
    const float alpha = expf(mx - nm);  // mx = -inf on the first tile: 0
    l *= alpha;
#pragma unroll
    for (int i = 0; i < DPT; ++i) acc[i] *= alpha;
#pragma unroll
    for (int r = 0; r < kTileRows; ++r) {
      if (r < nr) {
        const float p = expf(s[r] - nm);
        l += p;
#pragma unroll
        for (int c = 0; c < NV; ++c) {
          const float4 v4 = *reinterpret_cast<const float4*>(&Vs[r][(c * tpq + part) * 4]);
          acc[c * 4 + 0] += p * v4.x;
          acc[c * 4 + 1] += p * v4.y;
          acc[c * 4 + 2] += p * v4.z;
          acc[c * 4 + 3] += p * v4.w;
        }
      }
    }
    mx = nm;
  }
  if (!sum) return;
  // eta_N = log sum exp(s), m_N = sum exp(s - eta_N) v, merged with (eta_A, m_A)
  const float eta_n = mx + logf(l);
  const float inv_l = 1.f / l;
  float wa, wn, eta;
  if (eta_a == -INFINITY) {  // empty A: the merge returns N
    wa = 0.f; wn = inv_l; eta = eta_n;
  } else {
    const float mu = fmaxf(eta_a, eta_n);
    eta = mu + logf(expf(eta_a - mu) + expf(eta_n - mu));
    wa = expf(eta_a - eta);
    wn = expf(eta_n - eta) * inv_l;
  }
#pragma unroll
  for (int c = 0; c < NV; ++c) {
    const int dim = (c * tpq + part) * 4;
    const float4 m_a = wa != 0.f ? ma[c] : make_float4(0.f, 0.f, 0.f, 0.f);
    float4 r;
    r.x = wa * m_a.x + wn * acc[c * 4 + 0];
    r.y = wa * m_a.y + wn * acc[c * 4 + 1];
    r.z = wa * m_a.z + wn * acc[c * 4 + 2];
    r.w = wa * m_a.w + wn * acc[c * 4 + 3];
    *reinterpret_cast<float4*>(Mq + dim) = r;
  }
  if (part == 0) *etaq = eta;
}

template <typename T, int DPT>
__global__ void __launch_bounds__(kThreads) views_update_kernel(UpdateArgs a) {
  views_update_body<T, DPT>(a);
  commit_tail(a.ct);
}

// bf16 path on the matrix cores (v_mfma_f32_16x16x32_bf16). One wave per 16
// summary queries of the group (NW = rep * R / 16 waves); per tile of up to 32
// new rows, K rows (row-major) and V^T go to LDS as bf16, then
//  * S = G K^T on the matrix cores: bf16 products are exact in fp32 and the
//    sums are fp32, as on the vector path;
//  * the online log-sum-exp per query in fp32 (row max and sum over the 16
//    lanes of a C-layout row group with DPP);
//  * O += P V with P split into two bf16 terms, hi = bf16(P) and
//    lo = bf16(P - hi), so P enters with a relative error near 2^-17 rather
//    than bf16's 2^-9 (two MFMAs per tile instead of one);
// then the merge of Eq. 11 with the stored (eta, m), as on the vector path.
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ inline bf16x8 frag8(const uint16_t* p) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(p));
}
__device__ inline void wave_lds_fence() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

template <int DH, int NW>
__device__ __forceinline__ void views_update_mfma_body(const UpdateArgs& a) {
  constexpr int KT = 32, KS = DH / 32, NT = DH / 16, NTH = NW * 64;
  constexpr int KLD = DH + 8, VLD = KT + 8;   // padded LDS rows (elements)
  __shared__ __attribute__((aligned(16))) uint16_t Kt[KT * KLD];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[DH * VLD];
  __shared__ __attribute__((aligned(16))) uint16_t Pt[NW][2][16 * VLD];
  const int g = blockIdx.x, j = blockIdx.y, b = blockIdx.z;
  const int n = a.n_new[b];
  if (n <= 0 || n > a.max_new) return;  // empty set: identity; bad count: commit flags it
  const int64_t t = a.pos[b];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  uint8_t* seq = a.arena + (size_t)b * a.stride;

  // the wave's queries: rows q0 .. q0 + 15 of G, M and eta (C layout: this
  // lane holds rows q0 + lg * 4 + v, dims dt * 16 + lr)
  const size_t q0 = ((size_t)j * a.hq + (size_t)g * a.rep) * a.R + (size_t)wave * 16;
  float* Mq = reinterpret_cast<float*>(seq + a.m) + q0 * DH;
  float* etaq = reinterpret_cast<float*>(seq + a.eta) + q0;
  const bool sum = a.keep_sum, win = a.keep_win;
  float ma[NT][4], eta_a[4];
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    eta_a[v] = sum ? etaq[lg * 4 + v] : -INFINITY;
#pragma unroll
    for (int dt = 0; dt < NT; ++dt)
      ma[dt][v] = sum ? Mq[(size_t)(lg * 4 + v) * DH + dt * 16 + lr] : 0.f;
  }
  bf16x8 gf[KS];   // A layout: query row lr, dims ks * 32 + lg * 8 ..
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) gf[ks] = bf16x8{};
  if (sum) {
    const uint16_t* Gq = static_cast<const uint16_t*>(a.G) + (q0 + lr) * DH + lg * 8;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) gf[ks] = frag8(Gq + ks * 32);
  }

  if (a.keep_bnd) boundary_slice<uint16_t>(a, seq, j, g, b, NTH);

  uint16_t* Kw = reinterpret_cast<uint16_t*>(seq + a.kw) + ((size_t)(j * a.hkv + g) * a.Wx) * DH;
  uint16_t* Vw = reinterpret_cast<uint16_t*>(seq + a.vw) + ((size_t)(j * a.hkv + g) * a.Wx) * DH;
  const uint16_t* Kn = static_cast<const uint16_t*>(a.K_new);
  const uint16_t* Vn = static_cast<const uint16_t*>(a.V_new);
  f32x4 o[NT];
#pragma unroll
  for (int dt = 0; dt < NT; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m[4], l[4];
#pragma unroll
  for (int v = 0; v < 4; ++v) { m[v] = -INFINITY; l[v] = 0.f; }

  for (int r0 = 0; r0 < ((win || sum) ? n : 0); r0 += KT) {
    const int nr = min(KT, n - r0);
    __syncthreads();   // the previous tile's LDS reads are done
    // stage the tile (rows past nr as zeros) and ring-write the K rows that survive
    for (int i = tid; i < KT * (DH / 8); i += NTH) {
      const int r = i / (DH / 8), c8 = (i % (DH / 8)) * 8;
      u32x4 kv = u32x4{0u, 0u, 0u, 0u}, vv = kv;
      if (r < nr) {
        const size_t src = ((((size_t)b * a.max_new + r0 + r) * a.D + j) * a.hkv + g) * DH + c8;
        kv = *reinterpret_cast<const u32x4*>(Kn + src);
        vv = *reinterpret_cast<const u32x4*>(Vn + src);
        if (win && r0 + r >= n - a.W) {
          const size_t slot = (size_t)((t + r0 + r) % a.W);
          *reinterpret_cast<u32x4*>(Kw + slot * DH + c8) = kv;
        }
      }
      *reinterpret_cast<u32x4*>(&Kt[r * KLD + c8]) = kv;
      const uint16_t* vp = reinterpret_cast<const uint16_t*>(&vv);
#pragma unroll
      for (int e = 0; e < 8; ++e) Vt[(c8 + e) * VLD + r] = vp[e];
    }
    __syncthreads();
    {  // window V^T: lanes take consecutive rows of one dim (contiguous slots)
      const int rs = max(0, n - a.W - r0);
      const int r = tid % KT;
      if (win && r >= rs && r < nr) {
        const size_t slot = (size_t)((t + r0 + r) % a.W);
        for (int e = tid / KT; e < DH; e += NTH / KT) Vw[(size_t)e * a.Wx + slot] = Vt[e * VLD + r];
      }
    }
    if (!sum) continue;   // window only: no statistics
    // scores of keys nt * 16 + lr (C layout), scaled; keys past nr masked
    f32x4 sc[2];
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      sc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        sc[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
            gf[ks], frag8(&Kt[(nt * 16 + lr) * KLD + ks * 32 + lg * 8]), sc[nt], 0, 0, 0);
    }
    uint16_t* Ph = Pt[wave][0];
    uint16_t* Pl = Pt[wave][1];
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const float x0 = lr < nr ? sc[0][v] * a.inv_sqrt_d : -INFINITY;
      const float x1 = 16 + lr < nr ? sc[1][v] * a.inv_sqrt_d : -INFINITY;
      const float mn = fmaxf(m[v], max16(fmaxf(x0, x1)));
      const float alpha = expf(m[v] - mn);   // m = -inf on the first tile: 0
      const float p0 = expf(x0 - mn), p1 = expf(x1 - mn);
      l[v] = l[v] * alpha + sum16(p0 + p1);
      m[v] = mn;
#pragma unroll
      for (int dt = 0; dt < NT; ++dt) o[dt][v] *= alpha;
      const uint16_t h0 = f32_to_bf16(p0), h1 = f32_to_bf16(p1);
      const int row = (lg * 4 + v) * VLD;
      Ph[row + lr] = h0;
      Ph[row + 16 + lr] = h1;
      Pl[row + lr] = f32_to_bf16(p0 - bf16_to_f32(h0));
      Pl[row + 16 + lr] = f32_to_bf16(p1 - bf16_to_f32(h1));
    }
    wave_lds_fence();
    const bf16x8 phi = frag8(&Ph[lr * VLD + lg * 8]);
    const bf16x8 plo = frag8(&Pl[lr * VLD + lg * 8]);
#pragma unroll
    for (int dt = 0; dt < NT; ++dt) {
      const bf16x8 vf = frag8(&Vt[(dt * 16 + lr) * VLD + lg * 8]);
      o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(phi, vf, o[dt], 0, 0, 0);
      o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(plo, vf, o[dt], 0, 0, 0);
    }
  }
  if (!sum) return;
  // eta_N = m + log l, m_N = O / l, merged with (eta_A, m_A) (Eq. 11)
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const float eta_n = m[v] + logf(l[v]);
    const float inv_l = 1.f / l[v];
    float wa, wn, e;
    if (eta_a[v] == -INFINITY) {  // empty A: the merge returns N
      wa = 0.f; wn = inv_l; e = eta_n;
    } else {
      const float mu = fmaxf(eta_a[v], eta_n);
      e = mu + logf(expf(eta_a[v] - mu) + expf(eta_n - mu));
      wa = expf(eta_a[v] - e);
      wn = expf(eta_n - e) * inv_l;
    }
#pragma unroll
    for (int dt = 0; dt < NT; ++dt) {
      const float mav = wa != 0.f ? ma[dt][v] : 0.f;
      Mq[(size_t)(lg * 4 + v) * DH + dt * 16 + lr] = wa * mav + wn * o[dt][v];
    }
    if (lr == 0) etaq[lg * 4 + v] = e;
  }
}

template <int DH, int NW>
__global__ void __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(3)))
views_update_mfma_kernel(UpdateArgs a) {
  views_update_mfma_body<DH, NW>(a);
  commit_tail(a.ct);
}

// Mean-pooled summary (the views as the configurations word them): for each
// of two strides S, slot c mod P of the bank holds the mean K and V row of
// chunk c = rows [cS, (c+1)S). One workgroup per (kv group, layer, sequence);
// thread (bank, e) owns dim e of one bank. The chunks the new rows touch are
// summed in fp32 in row order, the open chunk continuing from its stored sums,
// and each slot takes sum / rows so far; only the last P chunks are written
// (older ones would be recycled by the same update). Slots are the bank rows
// after the window rows of the (layer, group) region: K row-major, V
// transposed, like the window.
struct PoolArgs {
  uint8_t* arena; size_t stride, kw, vw, ps;
  const int64_t* pos; const int32_t* n_new; int max_new;
  const void* K_new; const void* V_new;
  int D, hkv, d, Wr, Wx, P, S0, S1;
  CommitTail ct;
};

template <typename T>
__device__ __forceinline__ void views_pool_body(const PoolArgs& a) {
  const int g = blockIdx.x, j = blockIdx.y, b = blockIdx.z;
  const int n = a.n_new[b];
  if (n <= 0 || n > a.max_new) return;   // empty set: identity; bad count: commit flags it
  const int d = a.d, bank = (int)threadIdx.x / d, e = (int)threadIdx.x % d;
  const int64_t t = a.pos[b], S = bank ? a.S1 : a.S0;
  uint8_t* seq = a.arena + (size_t)b * a.stride;
  const size_t grp = (size_t)j * a.hkv + g;
  T* Kw = reinterpret_cast<T*>(seq + a.kw) + grp * a.Wx * d;
  T* Vw = reinterpret_cast<T*>(seq + a.vw) + grp * a.Wx * d;
  float* ps = reinterpret_cast<float*>(seq + a.ps) + (grp * 2 + bank) * 2 * d;   // K sums, V sums
  const T* Kn = static_cast<const T*>(a.K_new);
  const T* Vn = static_cast<const T*>(a.V_new);
  const int64_t c0 = t / S, c1 = (t + n - 1) / S;
  const int64_t cfirst = c0 > c1 - a.P + 1 ? c0 : c1 - a.P + 1;
  float sk = 0.f, sv = 0.f;
  for (int64_t c = cfirst; c <= c1; ++c) {
    const int64_t r0 = t > c * S ? t : c * S, r1 = t + n < (c + 1) * S ? t + n : (c + 1) * S;
    const bool carry = c == c0 && t % S != 0;   // the chunk was opened by an earlier update
    sk = carry ? ps[e] : 0.f;
    sv = carry ? ps[d + e] : 0.f;
    for (int64_t p = r0; p < r1; ++p) {
      const size_t src = ((((size_t)b * a.max_new + (size_t)(p - t)) * a.D + j) * a.hkv + g) * d + e;
      sk += Elem<T>::load(Kn + src);
      sv += Elem<T>::load(Vn + src);
    }
    const float cnt = (float)(r1 - c * S);
    const int slot = a.Wr + bank * a.P + (int)(c % a.P);
    Elem<T>::store(Kw + (size_t)slot * d + e, sk / cnt);
    Elem<T>::store(Vw + (size_t)e * a.Wx + slot, sv / cnt);
  }
  ps[e] = sk;   // the last chunk's sums (used next time only if it is still open)
  ps[d + e] = sv;
}

template <typename T>
__global__ void __launch_bounds__(256) views_pool_kernel(PoolArgs a) {
  views_pool_body<T>(a);
  commit_tail(a.ct);
}

__global__ void views_commit_kernel(int batch, int64_t* pos, const int32_t* n_new,
                                    int max_new, int32_t* status) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= batch) return;
  const int n = n_new[b];
  if (n < 0 || n > max_new)
    atomicOr(status, kFlagRange);
  else
    pos[b] += n;
}

template <typename T>
hipError_t launch_update_t(const UpdateArgs& a, int dpt, dim3 grid, hipStream_t st) {
  switch (dpt) {
    case 4: hipLaunchKernelGGL((views_update_kernel<T, 4>), grid, dim3(kThreads), 0, st, a); break;
    case 8: hipLaunchKernelGGL((views_update_kernel<T, 8>), grid, dim3(kThreads), 0, st, a); break;
    case 16: hipLaunchKernelGGL((views_update_kernel<T, 16>), grid, dim3(kThreads), 0, st, a); break;
    case 32: hipLaunchKernelGGL((views_update_kernel<T, 32>), grid, dim3(kThreads), 0, st, a); break;
    case 64: hipLaunchKernelGGL((views_update_kernel<T, 64>), grid, dim3(kThreads), 0, st, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

// Threads per summary query: Q = rep * R queries share 256 threads.
int views_dims_per_thread(const Shape& s) {
  if (s.R == 0) return s.d % 16 == 0 ? 16 : 0;   // no learned queries: ring writes only
  const int q = s.rep * s.R;
  if (q <= 0 || q > kThreads || kThreads % q) return 0;
  const int tpq = kThreads / q;
  if (tpq > 64 || s.d % tpq || s.d > 256) return 0;
  const int dpt = s.d / tpq;
  return (dpt == 4 || dpt == 8 || dpt == 16 || dpt == 32 || dpt == 64) ? dpt : 0;
}

hipError_t launch_views_reset(const Shape& s, const Layout& L, int batch, void* arena,
                              int64_t* pos, hipStream_t st) {
  const size_t words = L.stride / 4 * (size_t)batch;
  const int blocks = (int)((words + kThreads - 1) / kThreads < 4096
                               ? (words + kThreads - 1) / kThreads : 4096);
  const size_t eta_bytes = s.learned ? (size_t)s.D * s.hq * s.R * 4 : 0;
  hipLaunchKernelGGL(views_reset_kernel, dim3(blocks > 0 ? blocks : 1), dim3(kThreads), 0, st,
                     static_cast<uint8_t*>(arena), L.stride, L.eta, eta_bytes, batch, pos);
  return hipGetLastError();
}

hipError_t launch_views_update(const Shape& s, const Layout& L, int batch, void* arena,
                               int64_t* pos, const void* G, const int32_t* n_new,
                               int max_new, const void* K_new, const void* V_new,
                               const void* h_new, hipStream_t st, int32_t* status,
                               int32_t* done) {
  UpdateArgs a;
  a.arena = static_cast<uint8_t*>(arena); a.stride = L.stride;
  a.kw = L.kw; a.vw = L.vw; a.m = L.m; a.eta = L.eta; a.h = L.h;
  a.pos = pos; a.G = G; a.n_new = n_new; a.max_new = max_new;
  a.K_new = K_new; a.V_new = V_new; a.h_new = h_new;
  a.D = s.D; a.hq = s.hq; a.hkv = s.hkv; a.d = s.d; a.W = s.W; a.R = s.R; a.rep = s.rep;
  a.hb_elems = s.Lb * s.hidden;
  a.keep_win = s.keep_win; a.keep_sum = s.learned; a.keep_bnd = s.keep_bnd;
  a.Wx = s.Wx;
  a.inv_sqrt_d = 1.0f / sqrtf((float)s.d);
  const dim3 grid(s.hkv, s.D, batch);
  a.ct = CommitTail{done, (int)(grid.x * grid.y * grid.z), pos, n_new,
                    max_new, batch, status};
  const int q = s.rep * s.R;
  if (s.dtype == LDR_BF16 && (s.d == 64 || s.d == 128) && q % 16 == 0) {
    const int nw = q / 16;
#define LDR_VU(DH, NW) \
  if (s.d == DH && nw == NW) { \
    hipLaunchKernelGGL((views_update_mfma_kernel<DH, NW>), grid, dim3(NW * 64), 0, st, a); \
    return hipGetLastError(); \
  }
    LDR_VU(128, 4) LDR_VU(128, 2) LDR_VU(128, 8) LDR_VU(64, 4) LDR_VU(64, 2) LDR_VU(64, 8)
#undef LDR_VU
  }
  const int dpt = views_dims_per_thread(s);
  return s.dtype == LDR_BF16 ? launch_update_t<uint16_t>(a, dpt, grid, st)
                             : launch_update_t<float>(a, dpt, grid, st);
}

hipError_t launch_views_pool(const Shape& s, const Layout& L, int batch, void* arena,
                             int64_t* pos, const int32_t* n_new, int max_new,
                             const void* K_new, const void* V_new, hipStream_t st,
                             int32_t* status, int32_t* done) {
  PoolArgs a;
  a.arena = static_cast<uint8_t*>(arena); a.stride = L.stride; a.kw = L.kw; a.vw = L.vw;
  a.ps = L.ps; a.pos = pos; a.n_new = n_new; a.max_new = max_new; a.K_new = K_new;
  a.V_new = V_new; a.D = s.D; a.hkv = s.hkv; a.d = s.d; a.Wr = s.Wr; a.Wx = s.Wx; a.P = s.P;
  a.S0 = s.S0; a.S1 = s.S1;
  const dim3 grid(s.hkv, s.D, batch), block(2 * s.d);   // d <= 128
  a.ct = CommitTail{done, (int)(grid.x * grid.y * grid.z), pos, n_new,
                    max_new, batch, status};
  if (s.dtype == LDR_BF16)
    hipLaunchKernelGGL(views_pool_kernel<uint16_t>, grid, block, 0, st, a);
  else
    hipLaunchKernelGGL(views_pool_kernel<float>, grid, block, 0, st, a);
  return hipGetLastError();
}

hipError_t launch_views_commit(int batch, int64_t* pos, const int32_t* n_new, int max_new,
                               int32_t* status, hipStream_t st) {
  hipLaunchKernelGGL(views_commit_kernel, dim3((batch + 255) / 256), dim3(256), 0, st, batch,
                     pos, n_new, max_new, status);
  return hipGetLastError();
}

}  // namespace ldr
