// Speculative verification of a drafted block (Eq. 1-2): the consumer that
// closes a round.
//
// The target scores [a, y_1 .. y_B] in one pass, so sequence b brings B + 1
// rows of fp32 target logits P (row i is p_{i+1}); the draft brings its B rows
// of logits z (the proposal q_i = softmax(z_i / T), over the whole vocabulary)
// and the lse of each row from the sampler. Candidate y_i is accepted when
// u_i < p_i(y_i) / q_i(y_i), in order; the round then emits one token: at the
// first rejection a draw from [p_i - q_i]_+ normalised, after B acceptances a
// bonus draw from p_{B+1}. r accepted candidates advance the prefix by r + 1,
// which is the row count the next views update takes.
//
// Four launches at T > 0:
//  1. lse pass: one workgroup per (vocabulary chunk, candidate row) streams the
//     B target rows of every sequence once (16-byte loads) and writes the
//     chunk's running max and sum of exp(P / T);
//  2. decide: one wave per sequence merges the lse partials, takes the
//     in-order acceptance test (B exponentials) and writes r, r + 1 and the
//     normalisers of the row where the round stops;
//  3. emit pass: one workgroup per (sequence, vocabulary chunk) streams that
//     target row (and draft row, 16-byte loads): Gumbel keys log w_v + g_v
//     over the residual w = [p - q]_+ (every entry with w_v > 0 in fp32), and
//     the bonus-rule keys fl(fl(P_v / T) + g_v) (the draw at a bonus, and the
//     fallback when the residual has no positive mass);
//  4. merge: the best key over the chunks, lower token first on ties.
// T = 0 verifies greedily: pass 1 takes the first argmax of all B + 1 rows and
// the merge compares them with the candidates.
// A top-k proposal (the sampler's support, top_k > 0) has q = 0 outside the
// support: a selection pass finds each draft row's support first; a candidate
// outside it is rejected, and the residual there is p itself.
//
// Noise (the sampler's Philox4x32-10 layout): u_i is word 0 of block i - 1 of
// row b in stream 1; the emitted token's Gumbel noise is token v of row b in
// stream 2.
#include "ldr_internal.h"
#include "noise.h"

namespace ldr {
namespace {

constexpr int kThreads = 256;
constexpr int kInvalid = 0x7fffffff;

struct LsePart { float m, s; int idx, pad; };     // max P / T, sum exp(P / T - m); argmax at T = 0
struct EmitPart { float kr; int ir; float kb; int ib; };  // best residual key / bonus-rule key
struct Decision { int stop; float plse, qlse; int pad; };  // where a sequence stops, its normalisers

__device__ inline bool better(float k1, int i1, float k2, int i2) {
  return k1 > k2 || (k1 == k2 && i1 < i2);
}

__device__ inline void lse_combine(LsePart& a, const LsePart& b) {
  const float m = fmaxf(a.m, b.m);
  if (m == -INFINITY) return;
  a.s = a.s * __expf(a.m - m) + b.s * __expf(b.m - m);
  a.m = m;
}

// greedy: m holds the best logit, idx its first token
__device__ inline void max_combine(LsePart& a, const LsePart& b) {
  if (better(b.m, b.idx, a.m, a.idx)) { a.m = b.m; a.idx = b.idx; }
}

struct VerifyArgs {
  const float* P;        // [batch][B + 1][V]
  const float* z;        // [batch][B][V]
  const int32_t* y;      // [batch][B]
  const float* qlse;     // [batch][B]
  const TopK* sel;       // [batch][B] top-k support of the draft rows, or null (all tokens)
  int batch, B, V;
  float T;
  uint64_t seed, step;
  int chunk1, splits1;   // lse pass: rows of B (T > 0) or B + 1 (T = 0) per sequence
  int chunk2, splits2;   // emit pass
  LsePart* lpart;        // [batch * rows][splits1]
  EmitPart* epart;       // [batch][splits2]
  Decision* dec;         // [batch]
  int32_t* accepted; int32_t* token; int32_t* n_new;
};

template <bool GREEDY, bool VEC>
__global__ void __launch_bounds__(kThreads) verify_lse_kernel(VerifyArgs a) {
  const int row = blockIdx.x, sp = blockIdx.y;   // row: b * rows + i
  const int rows = GREEDY ? a.B + 1 : a.B;
  const int b = row / rows, i = row - b * rows;
  const float* p = a.P + ((long)b * (a.B + 1) + i) * a.V;
  const int v0 = sp * a.chunk1, v1 = min(a.V, v0 + a.chunk1);
  const float invT = GREEDY ? 1.f : 1.f / a.T;   // lse only: a product is close enough
  LsePart acc{-INFINITY, 0.f, kInvalid, 0};
  auto take1 = [&](float x, int v) {   // greedy: first maximum
    if (better(x, v, acc.m, acc.idx)) { acc.m = x; acc.idx = v; }
  };
  auto take4 = [&](float4 x) {          // T > 0: running max and sum of exp(P / T)
    const float t0 = x.x * invT, t1 = x.y * invT, t2 = x.z * invT, t3 = x.w * invT;
    const float mx = fmaxf(fmaxf(t0, t1), fmaxf(t2, t3));
    if (mx == -INFINITY) return;        // all four are -inf: nothing to add
    if (mx > acc.m) { acc.s *= __expf(acc.m - mx); acc.m = mx; }
    acc.s += __expf(t0 - acc.m) + __expf(t1 - acc.m) + __expf(t2 - acc.m) + __expf(t3 - acc.m);
  };
  if constexpr (VEC) {   // V % 4 == 0: chunks hold whole float4s; 4 loads in flight
    constexpr int U = 4;
    for (int v = v0 + 4 * (int)threadIdx.x; v < v1; v += 4 * kThreads * U) {
      float4 x[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int vu = v + u * 4 * kThreads;
        x[u] = vu < v1 ? *reinterpret_cast<const float4*>(p + vu)
                       : float4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int vu = v + u * 4 * kThreads;
        if constexpr (GREEDY) {
          if (vu < v1) {
            take1(x[u].x, vu); take1(x[u].y, vu + 1); take1(x[u].z, vu + 2); take1(x[u].w, vu + 3);
          }
        } else {
          take4(x[u]);
        }
      }
    }
  } else {
    for (int v = v0 + (int)threadIdx.x; v < v1; v += kThreads) {
      if constexpr (GREEDY) take1(p[v], v);
      else take4(float4{p[v], -INFINITY, -INFINITY, -INFINITY});
    }
  }
  for (int off = 32; off >= 1; off >>= 1) {
    LsePart o{__shfl_xor(acc.m, off), __shfl_xor(acc.s, off), __shfl_xor(acc.idx, off), 0};
    if constexpr (GREEDY) max_combine(acc, o); else lse_combine(acc, o);
  }
  __shared__ LsePart red[kThreads / 64];
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < kThreads / 64; ++w) {
      if constexpr (GREEDY) max_combine(acc, red[w]); else lse_combine(acc, red[w]);
    }
    a.lpart[(long)row * a.splits1 + sp] = acc;
  }
}

// log-normaliser of candidate row i of sequence b from the lse partials
__device__ inline float row_lse(const VerifyArgs& a, int b, int i) {
  const LsePart* q = a.lpart + ((long)b * a.B + i) * a.splits1;
  LsePart acc = q[0];
  for (int s = 1; s < a.splits1; ++s) lse_combine(acc, q[s]);
  return acc.m + logf(acc.s);
}

// Position where the round stops (B if every candidate passes), by the
// acceptance test of Eq. 1 on the lanes of one wave, 64 candidates at a time.
__device__ int stop_position(const VerifyArgs& a, int b) {
  const int lane = threadIdx.x & 63;
  for (int i0 = 0; i0 < a.B; i0 += 64) {
    const int i = i0 + lane;
    bool reject = false;
    if (i < a.B) {
      const int y = a.y[(long)b * a.B + i];
      const float* zi = a.z + ((long)b * a.B + i) * a.V;
      if (y < 0 || y >= a.V || (a.sel && !in_support(a.sel[(long)b * a.B + i], zi[y], y))) {
        reject = true;   // q(y) = 0: the proposal cannot produce y
      } else {
        const float lp = a.P[((long)b * (a.B + 1) + i) * a.V + y] / a.T - row_lse(a, b, i);
        const float lq = zi[y] / a.T - a.qlse[(long)b * a.B + i];
        const float ratio = expf(lp - lq);
        uint32_t w[4];
        noise_block(noise_key(a.seed, a.step, 1), (uint32_t)b, (uint32_t)i, w);
        reject = !(uniform_from_bits(w[0]) < ratio);
      }
    }
    const uint64_t m = __ballot(reject);
    if (m) return i0 + __ffsll((unsigned long long)m) - 1;
  }
  return a.B;
}

// One wave per sequence: the acceptance test, r and r + 1, and the
// normalisers of the row where the round stops.
__global__ void __launch_bounds__(64) verify_decide_kernel(VerifyArgs a) {
  const int b = blockIdx.x;
  const int stop = stop_position(a, b);
  if (threadIdx.x == 0) {
    Decision d{stop, 0.f, 0.f, 0};
    if (stop < a.B) { d.plse = row_lse(a, b, stop); d.qlse = a.qlse[(long)b * a.B + stop]; }
    a.dec[b] = d;
    a.accepted[b] = stop;
    a.n_new[b] = stop + 1;
  }
}

template <bool UNIT_T, bool VEC>
__global__ void __launch_bounds__(kThreads) verify_emit_kernel(VerifyArgs a) {
  const int b = blockIdx.x, sp = blockIdx.y;
  const Decision d = a.dec[b];
  const int stop = d.stop;
  const bool residual = stop < a.B;
  const float plse = d.plse, qlse = d.qlse;
  const float* p = a.P + ((long)b * (a.B + 1) + stop) * a.V;
  const float* z = residual ? a.z + ((long)b * a.B + stop) * a.V : nullptr;
  const TopK sel = residual && a.sel ? a.sel[(long)b * a.B + stop] : TopK{0u, -1};
  const int v0 = sp * a.chunk2, v1 = min(a.V, v0 + a.chunk2);
  EmitPart e{-INFINITY, kInvalid, -INFINITY, kInvalid};
  // A token's exact keys (two logarithms for g, more for the residual) are
  // computed only where an upper bound from the noise bits cannot rule them
  // out: g <= gumbel_upper(bits), so kb <= pt + bound and, as w <= p,
  // kr <= pt - plse + bound. The bounds are tested against the best keys of
  // the whole wave so far, seeded in each sweep by the exact keys of every
  // lane's largest logit. The margin covers the rounding of the bound and of
  // the exact keys: a token skipped has a key strictly below the best.
  auto exact = [&](int v, float pt, float zv, uint32_t word, bool want_b, bool want_r) {
    const float g = gumbel_from_bits(word);
    if (want_b) {
      const float kb = __fadd_rn(pt, g);
      if (better(kb, v, e.kb, e.ib)) { e.kb = kb; e.ib = v; }
    }
    if (want_r) {
      const float zt = UNIT_T ? zv : zv / a.T;
      const float pv = expf(pt - plse);
      // q = 0 outside a top-k support (the whole vocabulary has tau = 0)
      const float qv = in_support(sel, zv, v) ? expf(zt - qlse) : 0.f;
      const float w = pv - qv;
      if (w > 0.f) {   // Eq. 2: [p - q]_+
        const float kr = logf(w) + g;
        if (better(kr, v, e.kr, e.ir)) { e.kr = kr; e.ir = v; }
      }
    }
  };
  for (int vb0 = v0; vb0 < v1; vb0 += kThreads * kGroup) {
    const int vb = vb0 + (int)threadIdx.x * kGroup;
    uint32_t bits[kGroup];
    noise_group(a.seed, a.step, (uint64_t)b, 2, (uint64_t)(vb / kGroup), bits);
    float pr[kGroup], zr[kGroup];
    if (VEC && vb + kGroup <= v1) {   // 16-byte aligned: V % 4 == 0 and vb % 8 == 0
      const float4 p0 = *reinterpret_cast<const float4*>(p + vb);
      const float4 p1 = *reinterpret_cast<const float4*>(p + vb + 4);
      pr[0] = p0.x; pr[1] = p0.y; pr[2] = p0.z; pr[3] = p0.w;
      pr[4] = p1.x; pr[5] = p1.y; pr[6] = p1.z; pr[7] = p1.w;
      if (residual) {
        const float4 z0 = *reinterpret_cast<const float4*>(z + vb);
        const float4 z1 = *reinterpret_cast<const float4*>(z + vb + 4);
        zr[0] = z0.x; zr[1] = z0.y; zr[2] = z0.z; zr[3] = z0.w;
        zr[4] = z1.x; zr[5] = z1.y; zr[6] = z1.z; zr[7] = z1.w;
      }
    } else {
#pragma unroll
      for (int k = 0; k < kGroup; ++k) {
        pr[k] = vb + k < v1 ? p[vb + k] : -INFINITY;
        zr[k] = residual && vb + k < v1 ? z[vb + k] : 0.f;
      }
    }
    float pt[kGroup];
    int km = 0;
#pragma unroll
    for (int k = 0; k < kGroup; ++k) {
      pt[k] = UNIT_T ? pr[k] : pr[k] / a.T;   // IEEE division, as the drafting sampler
      if (pt[k] > pt[km]) km = k;
    }
    // seed: the exact keys of the lane's largest logit, then the wave's best
    if (vb + km < v1) {
      float zkm = zr[0];
      uint32_t wkm = bits[0];
#pragma unroll
      for (int k = 1; k < kGroup; ++k)
        if (k == km) { zkm = zr[k]; wkm = bits[k]; }
      exact(vb + km, pt[km], zkm, wkm, true, residual);
    }
    float tb = e.kb, tr = e.kr;
    for (int off = 32; off >= 1; off >>= 1) {
      tb = fmaxf(tb, __shfl_xor(tb, off));
      tr = fmaxf(tr, __shfl_xor(tr, off));
    }
#pragma unroll
    for (int k = 0; k < kGroup; ++k) {
      const int v = vb + k;
      if (v >= v1 || k == km) continue;
      const float gu = gumbel_upper(bits[k]);
      const bool need_b = !(pt[k] + gu + (1e-3f + 1e-6f * (fabsf(pt[k]) + fabsf(tb))) < tb);
      const float lp = pt[k] - plse;
      const bool need_r = residual && !(lp + gu + (1e-3f + 1e-6f * (fabsf(lp) + fabsf(tr))) < tr);
      if (need_b || need_r) exact(v, pt[k], zr[k], bits[k], need_b, need_r);
    }
  }
  for (int off = 32; off >= 1; off >>= 1) {
    const EmitPart o{__shfl_xor(e.kr, off), __shfl_xor(e.ir, off), __shfl_xor(e.kb, off),
                     __shfl_xor(e.ib, off)};
    if (better(o.kr, o.ir, e.kr, e.ir)) { e.kr = o.kr; e.ir = o.ir; }
    if (better(o.kb, o.ib, e.kb, e.ib)) { e.kb = o.kb; e.ib = o.ib; }
  }
  __shared__ EmitPart red[kThreads / 64];
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = e;
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < kThreads / 64; ++w) {
      const EmitPart& o = red[w];
      if (better(o.kr, o.ir, e.kr, e.ir)) { e.kr = o.kr; e.ir = o.ir; }
      if (better(o.kb, o.ib, e.kb, e.ib)) { e.kb = o.kb; e.ib = o.ib; }
    }
    a.epart[(long)b * a.splits2 + sp] = e;
  }
}

__global__ void __launch_bounds__(64) verify_merge_kernel(VerifyArgs a) {
  const int b = blockIdx.x;
  EmitPart e{-INFINITY, kInvalid, -INFINITY, kInvalid};
  for (int s = threadIdx.x; s < a.splits2; s += 64) {
    const EmitPart& o = a.epart[(long)b * a.splits2 + s];
    if (better(o.kr, o.ir, e.kr, e.ir)) { e.kr = o.kr; e.ir = o.ir; }
    if (better(o.kb, o.ib, e.kb, e.ib)) { e.kb = o.kb; e.ib = o.ib; }
  }
  for (int off = 32; off >= 1; off >>= 1) {
    const EmitPart o{__shfl_xor(e.kr, off), __shfl_xor(e.ir, off), __shfl_xor(e.kb, off),
                     __shfl_xor(e.ib, off)};
    if (better(o.kr, o.ir, e.kr, e.ir)) { e.kr = o.kr; e.ir = o.ir; }
    if (better(o.kb, o.ib, e.kb, e.ib)) { e.kb = o.kb; e.ib = o.ib; }
  }
  // a residual without positive mass (or a bonus) takes the bonus-rule draw
  if (threadIdx.x == 0) a.token[b] = e.ir != kInvalid ? e.ir : e.ib;
}

// T = 0: the first argmax of each of the B + 1 rows, then the longest run of
// candidates equal to them.
__global__ void __launch_bounds__(64) verify_greedy_kernel(VerifyArgs a) {
  const int b = blockIdx.x, lane = threadIdx.x;
  int stop = a.B, tok = 0;
  for (int i0 = 0; i0 <= a.B; i0 += 64) {
    const int i = i0 + lane;
    int best = kInvalid;
    bool reject = false;
    if (i <= a.B) {
      const LsePart* q = a.lpart + ((long)b * (a.B + 1) + i) * a.splits1;
      LsePart acc = q[0];
      for (int s = 1; s < a.splits1; ++s) max_combine(acc, q[s]);
      best = acc.idx;
      reject = i == a.B || a.y[(long)b * a.B + i] != best;   // row B always stops the run
    }
    const uint64_t m = __ballot(reject);
    if (m) {
      const int first = __ffsll((unsigned long long)m) - 1;
      stop = i0 + first;
      tok = __shfl(best, first);
      break;
    }
  }
  if (lane == 0) {
    a.accepted[b] = stop;
    a.n_new[b] = stop + 1;
    a.token[b] = tok;
  }
}

struct Plan { int chunk1, splits1, chunk2, splits2; };

Plan make_plan(int batch, int B, int V, bool greedy) {
  Plan p;
  const int rows = batch * (greedy ? B + 1 : B);
  // lse pass: about 2048 workgroups, chunks of whole 16-byte sweeps
  const int sweep1 = 4 * kThreads;
  int s1 = rows >= 2048 ? 1 : 2048 / rows;
  const int max1 = (V + sweep1 - 1) / sweep1;
  s1 = s1 < 1 ? 1 : (s1 > max1 ? max1 : s1);
  p.chunk1 = ((V + s1 - 1) / s1 + sweep1 - 1) / sweep1 * sweep1;
  p.splits1 = (V + p.chunk1 - 1) / p.chunk1;
  // emit pass: about 512 workgroups, chunks of whole Philox sweeps
  const int sweep2 = kGroup * kThreads;
  int s2 = batch >= 512 ? 1 : 512 / batch;
  const int max2 = (V + sweep2 - 1) / sweep2;
  s2 = s2 < 1 ? 1 : (s2 > max2 ? max2 : s2);
  p.chunk2 = ((V + s2 - 1) / s2 + sweep2 - 1) / sweep2 * sweep2;
  p.splits2 = (V + p.chunk2 - 1) / p.chunk2;
  return p;
}

}  // namespace

size_t verify_workspace_bytes(int batch, int B, int V) {
  const Plan g = make_plan(batch, B, V, true), t = make_plan(batch, B, V, false);
  const size_t l1 = (size_t)batch * (B + 1) * g.splits1, l2 = (size_t)batch * B * t.splits1;
  const size_t lse = align_up((l1 > l2 ? l1 : l2) * sizeof(LsePart));
  return lse + align_up((size_t)batch * t.splits2 * sizeof(EmitPart)) +
         align_up(batch * sizeof(Decision)) + (size_t)batch * B * sizeof(TopK);
}

hipError_t launch_verify(const float* P, const float* z, const int32_t* y, const float* qlse,
                         int batch, int B, int V, float T, int top_k, uint64_t seed,
                         uint64_t step, int32_t* accepted, int32_t* token, int32_t* n_new,
                         void* ws, hipStream_t st) {
  const bool greedy = T == 0.f;
  const Plan pl = make_plan(batch, B, V, greedy);
  VerifyArgs a;
  a.P = P; a.z = z; a.y = y; a.qlse = qlse;
  a.batch = batch; a.B = B; a.V = V; a.T = T; a.seed = seed; a.step = step;
  a.chunk1 = pl.chunk1; a.splits1 = pl.splits1; a.chunk2 = pl.chunk2; a.splits2 = pl.splits2;
  const Plan g = make_plan(batch, B, V, true), t = make_plan(batch, B, V, false);
  const size_t l1 = (size_t)batch * (B + 1) * g.splits1, l2 = (size_t)batch * B * t.splits1;
  a.lpart = static_cast<LsePart*>(ws);
  a.epart = reinterpret_cast<EmitPart*>(static_cast<uint8_t*>(ws) +
                                        align_up((l1 > l2 ? l1 : l2) * sizeof(LsePart)));
  a.dec = reinterpret_cast<Decision*>(reinterpret_cast<uint8_t*>(a.epart) +
                                      align_up((size_t)batch * pl.splits2 * sizeof(EmitPart)));
  a.accepted = accepted; a.token = token; a.n_new = n_new;
  a.sel = nullptr;
  if (!greedy && top_k > 0 && top_k < V && B > 0) {   // the draft rows' top-k supports
    TopK* sel = reinterpret_cast<TopK*>(reinterpret_cast<uint8_t*>(a.dec) +
                                        align_up(batch * sizeof(Decision)));
    const hipError_t e = launch_topk_select(z, batch * B, V, top_k, sel, st);
    if (e != hipSuccess) return e;
    a.sel = sel;
  }
  // 16-byte loads need rows that start on 16 bytes
  const bool vec = V % 4 == 0 && reinterpret_cast<uintptr_t>(P) % 16 == 0 &&
                   reinterpret_cast<uintptr_t>(z) % 16 == 0;
  const int rows = batch * (greedy ? B + 1 : B);
  const dim3 g1(rows, pl.splits1);
  if (greedy) {
    if (vec) hipLaunchKernelGGL((verify_lse_kernel<true, true>), g1, dim3(kThreads), 0, st, a);
    else hipLaunchKernelGGL((verify_lse_kernel<true, false>), g1, dim3(kThreads), 0, st, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(verify_greedy_kernel, dim3(batch), dim3(64), 0, st, a);
    return hipGetLastError();
  }
  if (B > 0) {
    if (vec) hipLaunchKernelGGL((verify_lse_kernel<false, true>), g1, dim3(kThreads), 0, st, a);
    else hipLaunchKernelGGL((verify_lse_kernel<false, false>), g1, dim3(kThreads), 0, st, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(verify_decide_kernel, dim3(batch), dim3(64), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const dim3 g2(batch, pl.splits2);
  if (T == 1.f) {
    if (vec) hipLaunchKernelGGL((verify_emit_kernel<true, true>), g2, dim3(kThreads), 0, st, a);
    else hipLaunchKernelGGL((verify_emit_kernel<true, false>), g2, dim3(kThreads), 0, st, a);
  } else {
    if (vec) hipLaunchKernelGGL((verify_emit_kernel<false, true>), g2, dim3(kThreads), 0, st, a);
    else hipLaunchKernelGGL((verify_emit_kernel<false, false>), g2, dim3(kThreads), 0, st, a);
  }
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(verify_merge_kernel, dim3(batch), dim3(64), 0, st, a);
  return hipGetLastError();
}

}  // namespace ldr
