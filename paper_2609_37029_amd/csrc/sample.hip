// Per-position sampling of the factorised proposal (Eq. 8).
//
// T > 0: a two-level Gumbel-max, an exact draw from q = softmax(z/T) over the
// support. The vocabulary is cut into chunks of 16 consecutive tokens; chunk c
// has log-mass L_c = log sum_{v in c} exp(z_v/T). The chunk is the first
// argmax of L_c + h_c (h_c Gumbel noise of stream 3), the token the first
// argmax of z_v/T + g_v over that chunk (g_v Gumbel noise of stream 0):
//  * chunk_lse_kernel streams the logits once (16-byte loads, four sweeps in
//    flight per lane) and writes L_c: a lane holds 4 tokens of a chunk, the
//    chunk's max and sum of exp(z/T - max) are reduced over its 4 lanes with
//    DPP, in the balanced pairwise order (t0 + t1) + (t2 + t3), ... over the
//    chunk's tokens;
//  * chunk_draw_kernel, one workgroup per row, runs the Gumbel-max over the
//    row's L_c like a one-level sampler over V/16 entries: per lane the
//    running max / sum of exp(L_c) for the log-normaliser and the best key,
//    exact keys computed only for entries that a cheap upper bound of the
//    noise cannot rule out; it combines the lanes' results (lower index wins
//    ties), then draws the token inside the winning chunk, one lane per
//    token, and writes the token, lse and log q(y).
// T = 0 is the first argmax of the logits (sample_partial_kernel + merge).
//
// The noise is a pure function of (seed, step, stream, row, entry):
// Philox4x32-10 (Salmon et al., SC 2011; key = the seed, counter (entry / 4,
// row, step, stream)); one Philox block serves 4 consecutive entries, 32 bits
// each. The uniform u = (2 (bits >> 9) + 1) 2^-24 is exact, and
// g = -log(-log u) uses a log made of IEEE fp32 operations only (no
// contraction, correctly rounded division), so every key fl(x + g) is
// reproducible bit for bit.
#include <mutex>

#include "ldr_internal.h"
#include "noise.h"

namespace ldr {
namespace {

constexpr int kThreads = 256;

struct Partial { float m, s, key; int idx; };  // max z/T, sum exp(z/T - m), best key, token

__device__ inline bool better(float k1, int i1, float k2, int i2) {
  return k1 > k2 || (k1 == k2 && i1 < i2);
}

__device__ inline void combine(Partial& a, const Partial& b) {
  if (better(b.key, b.idx, a.key, a.idx)) { a.key = b.key; a.idx = b.idx; }
  const float m = fmaxf(a.m, b.m);
  if (m == -INFINITY) return;
  a.s = a.s * __expf(a.m - m) + b.s * __expf(b.m - m);
  a.m = m;
}

struct SampleArgs {
  const float* logits; int rows, vocab, chunk, splits;
  float T; uint64_t seed, step;
  Partial* part;
  const TopK* sel;  // top-k support per row, or null for the full vocabulary
  int row_mul, row_add;  // row r of the launch is logits row (and noise row) r * mul + add
  int vec;               // rows start on 16 bytes (V % 4 == 0, aligned logits): 16-byte loads
  float* L;              // chunk log-masses [rows][ldL] (T > 0)
  int ldL, nch;          // row stride of L (a multiple of 4) and chunks per row
};

constexpr int kChunk = 16;        // tokens per vocabulary chunk of the two-level draw
constexpr uint32_t kChunkStream = 3;

// Exact k-th largest logit of a row by radix selection on order_key (four
// 8-bit digits, most significant first, LDS histograms), then the index cut
// among the tokens equal to it. One workgroup per row.
constexpr int kSelThreads = 1024;
__global__ void __launch_bounds__(kSelThreads) topk_select_kernel(const float* logits, int vocab,
                                                                  int k, TopK* sel, int row_mul,
                                                                  int row_add) {
  const float* z = logits + ((long)blockIdx.x * row_mul + row_add) * vocab;
  __shared__ uint32_t hist[256];
  __shared__ uint32_t s_digit, s_above;
  __shared__ int wcount[kSelThreads / 64];
  __shared__ int s_base, s_cut;
  uint32_t prefix = 0u, mask = 0u, count_eq = 0u;
  int remaining = k;  // rank of the wanted value among the keys matching prefix
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    for (int i = threadIdx.x; i < 256; i += kSelThreads) hist[i] = 0u;
    __syncthreads();
    for (int v = threadIdx.x; v < vocab; v += kSelThreads) {
      const uint32_t u = order_key(z[v]);
      if ((u & mask) == prefix) atomicAdd(&hist[(u >> shift) & 0xFFu], 1u);
    }
    __syncthreads();
    if (threadIdx.x == 0) {  // the digit where the count from the top reaches `remaining`
      uint32_t cum = 0u;
      int d = 255;
      for (; d > 0; --d) {
        if (cum + hist[d] >= (uint32_t)remaining) break;
        cum += hist[d];
      }
      s_digit = (uint32_t)d;
      s_above = cum;
    }
    __syncthreads();
    const uint32_t d = s_digit;
    remaining -= (int)s_above;
    prefix |= d << shift;
    mask |= 0xFFu << shift;
    count_eq = hist[d];
    __syncthreads();
  }
  // `remaining` of the count_eq tokens equal to the k-th value are inside:
  // the lowest indices first
  int v_cut = vocab;
  if (remaining < (int)count_eq) {
    if (threadIdx.x == 0) { s_base = 0; s_cut = -1; }
    __syncthreads();
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    for (int v0 = 0; v0 < vocab; v0 += kSelThreads) {
      const int v = v0 + (int)threadIdx.x;
      const bool eq = v < vocab && order_key(z[v]) == prefix;
      const uint64_t ball = __ballot(eq);
      if (lane == 0) wcount[w] = __popcll(ball);
      __syncthreads();
      int rank = s_base + __popcll(ball & ((1ull << lane) - 1ull)) + 1;
      for (int i = 0; i < w; ++i) rank += wcount[i];
      if (eq && rank == remaining) s_cut = v;
      __syncthreads();
      if (threadIdx.x == 0)
        for (int i = 0; i < kSelThreads / 64; ++i) s_base += wcount[i];
      __syncthreads();
      if (s_cut >= 0) break;  // uniform: read after the barrier
    }
    v_cut = s_cut;
  }
  if (threadIdx.x == 0) sel[blockIdx.x] = TopK{prefix, v_cut};
}

// The lane's G values of a sweep at v (G a multiple of 4): 16-byte loads
// inside the range [.., v1) when vec, else one load per entry (-inf past v1).
template <int G>
__device__ inline void load_group(const float* z, int v, int v1, bool vec, float (&zz)[G]) {
  if (vec && v + G <= v1) {
#pragma unroll
    for (int b = 0; b < G / 4; ++b) {
      const float4 x = *reinterpret_cast<const float4*>(z + v + 4 * b);
      zz[4 * b] = x.x; zz[4 * b + 1] = x.y; zz[4 * b + 2] = x.z; zz[4 * b + 3] = x.w;
    }
  } else {
#pragma unroll
    for (int i = 0; i < G; ++i) zz[i] = v + i < v1 ? z[v + i] : -INFINITY;
  }
}

// Greedy steps (T = 0): the first argmax of the chunk, its logits streamed in
// the sampling sweeps' pattern (the next sweep's loads in flight).
__device__ void argmax_tokens(const SampleArgs& a, const float* z, int v0, int v1, Partial& p) {
  constexpr int kSweep = kThreads * kGroup;
  const int lane_off = (int)threadIdx.x * kGroup;
  float znext[kGroup];
  load_group(z, v0 + lane_off, v1, a.vec, znext);
  for (int vb = v0; vb < v1; vb += kSweep) {
    const int v = vb + lane_off;
    float zcur[kGroup];
#pragma unroll
    for (int i = 0; i < kGroup; ++i) zcur[i] = znext[i];
    if (vb + kSweep < v1) load_group(z, v + kSweep, v1, a.vec, znext);
#pragma unroll
    for (int i = 0; i < kGroup; ++i)
      if (v + i < v1 && better(zcur[i], v + i, p.key, p.idx)) { p.key = zcur[i]; p.idx = v + i; }
  }
}

// Gumbel-max over the chunk log-masses L_c of row r, entries [c0, c1). Every
// lane keeps the max / sum of exp(L_c) of its entries (so the row's lse is
// log sum_c exp(L_c)) and the best (key, chunk) of the entries it evaluated
// exactly. Per sweep of G entries a lane evaluates first the exact key of
// its entry with the largest upper bound L_c + bound(h_c); the largest key of
// the wave so far is then a lower bound of the row's best, and any other
// entry is a candidate only unless L_c + bound(h_c) + margin < that bound,
// which proves that its exact key loses (the margin, 1e-3 plus 1e-6
// relative, covers the rounding of the test and of the fixed-sequence log,
// whose error is below 1e-5 here). Chunks without support tokens
// (L_c = -inf) take no part. Candidates go through a per-wave queue in LDS so
// that their exact keys (two logs each) are computed 64 at a time by full
// waves. G entries per lane and sweep (a multiple of 4, the noise words of
// G / 4 Philox blocks): with 12, one sweep of 1024 lanes covers 12288 chunks,
// a 196K-token vocabulary.
template <int NT, int G = kGroup>
__device__ void chunk_keys(const SampleArgs& a, const float* Lr, int r, int c0, int c1,
                           Partial& p) {
  struct Cand { float zt; uint32_t bits; int v; };
  __shared__ Cand queue[NT / 64][128];
  const int lane = threadIdx.x & 63;
  Cand* q = queue[threadIdx.x >> 6];
  int qn = 0;  // wave-uniform queue length
  auto drain = [&](int count) {  // evaluate entries [0, count), count <= 64
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
    if (lane < count) {
      const Cand c = q[lane];
      const float key = __fadd_rn(c.zt, gumbel_from_bits(c.bits));
      if (better(key, c.v, p.key, p.idx)) { p.key = key; p.idx = c.v; }
    }
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
  };
  constexpr int kSweep = NT * G;
  const int lane_off = (int)threadIdx.x * G;
  const uint64_t nrow = (uint64_t)r * a.row_mul + a.row_add;
  float znext[G];
  load_group(Lr, c0 + lane_off, c1, true, znext);
  for (int vb = c0; vb < c1; vb += kSweep) {
    const int v = vb + lane_off;
    float zt[G];
#pragma unroll
    for (int i = 0; i < G; ++i) zt[i] = znext[i];
    if (vb + kSweep < c1) load_group(Lr, v + kSweep, c1, true, znext);
    uint32_t bits[G];
    noise_group(a.seed, a.step, nrow, kChunkStream, (uint64_t)(v / G), bits);
    float gm = -INFINITY, ub[G];
    bool in[G];
    int top = -1;
    float top_ub = -INFINITY;
#pragma unroll
    for (int i = 0; i < G; ++i) {
      in[i] = v + i < c1 && zt[i] > -INFINITY;
      gm = fmaxf(gm, in[i] ? zt[i] : -INFINITY);
      ub[i] = zt[i] + gumbel_upper(bits[i]);
      if (in[i] && (top < 0 || ub[i] > top_ub)) { top = i; top_ub = ub[i]; }
    }
    if (gm > p.m) { p.s *= __expf(p.m - gm); p.m = gm; }
    // the lane's most promising entry, exactly; then the wave's best key
    float zsel = 0.f;
    uint32_t bsel = 0u;
#pragma unroll
    for (int i = 0; i < G; ++i)
      if (i == top) { zsel = zt[i]; bsel = bits[i]; }
    if (top >= 0) {
      const float key = __fadd_rn(zsel, gumbel_from_bits(bsel));
      if (better(key, v + top, p.key, p.idx)) { p.key = key; p.idx = v + top; }
    }
    float bound = p.key;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) bound = fmaxf(bound, __shfl_xor(bound, off));
#pragma unroll
    for (int i = 0; i < G; ++i) {
      const bool valid = in[i];
      if (valid) p.s += __expf(zt[i] - p.m);
      const float margin = 1e-3f + 1e-6f * (fabsf(zt[i]) + fabsf(bound));
      const bool need = valid && i != top && !(ub[i] + margin < bound);
      const uint64_t mask = __ballot(need);
      if (need) {
        const int pos = qn + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
        q[pos] = Cand{zt[i], bits[i], v + i};
      }
      qn += __popcll(mask);
      if (qn >= 64) {
        drain(64);
        if (lane < qn - 64) q[lane] = q[64 + lane];
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
        __builtin_amdgcn_wave_barrier();
        qn -= 64;
      }
    }
  }
  if (qn > 0) drain(qn);
}

// Chunk log-masses of tokens [v0, v1) of one row (v0 a multiple of 16): each
// lane takes 4 consecutive tokens, so 4 lanes hold a chunk. Whole groups of U
// sweeps of kThreads * 4 tokens load without bounds checks (U loads in flight
// per lane), the rest one guarded sweep at a time. Writes L_c for the chunks
// it covers.
template <bool UNIT_T, bool TOPK, bool VEC>
__global__ void __launch_bounds__(kThreads) chunk_lse_kernel(SampleArgs a, int v_begin,
                                                             int v_end, int slice) {
  constexpr int U = 4, kSweep = kThreads * 4;
  const int r = blockIdx.y;
  const int v0 = v_begin + blockIdx.x * slice, v1 = min(v_end, v0 + slice);
  const float* z = a.logits + ((long)r * a.row_mul + a.row_add) * a.vocab;
  float* L = a.L + (long)r * a.ldL;
  const TopK sel = TOPK ? a.sel[r] : TopK{0u, 0};
  const float T = a.T;
  const int t4 = 4 * (int)threadIdx.x;
  // the chunk of the 4 tokens x at v (tokens at or past v1 are outside)
  auto chunk = [&](int v, const float (&x)[4]) {
    float zt[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      bool in = v + i < v1;
      if constexpr (TOPK) in = in && in_support(sel, x[i], v + i);
      zt[i] = in ? (UNIT_T ? x[i] : x[i] / T) : -INFINITY;  // IEEE division
    }
    float m = fmaxf(fmaxf(zt[0], zt[1]), fmaxf(zt[2], zt[3]));
    m = fmaxf(m, dpp<0xB1>(m));   // the chunk's 4 lanes
    m = fmaxf(m, dpp<0x4E>(m));
    float e[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) e[i] = chunk_term(zt[i], m);
    float sum = (e[0] + e[1]) + (e[2] + e[3]);
    sum += dpp<0xB1>(sum);
    sum += dpp<0x4E>(sum);
    if ((threadIdx.x & 3) == 0 && v < v1) L[v / kChunk] = chunk_log_mass(m, sum);
  };
  int vb = v0;
  for (; vb + U * kSweep <= v1; vb += U * kSweep) {
    float x[U][4];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const float* zp = z + vb + u * kSweep + t4;
      if constexpr (VEC) {
        const float4 t = *reinterpret_cast<const float4*>(zp);
        x[u][0] = t.x; x[u][1] = t.y; x[u][2] = t.z; x[u][3] = t.w;
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) x[u][i] = zp[i];
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) chunk(vb + u * kSweep + t4, x[u]);
  }
  for (; vb < v1; vb += kSweep) {
    const int v = vb + t4;
    float x[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) x[i] = v + i < v1 ? z[v + i] : -INFINITY;
    chunk(v, x);
  }
}

// The chunk keys and the in-chunk draw of one row (T > 0), one workgroup of
// kDrawThreads threads per row: the Gumbel-max over all its chunk log-masses
// (each lane a sweep or two of 8 entries), the lanes' partials combined (max /
// sum of exp(L) for lse, best key and chunk), then lanes 0 .. 15 of the first
// wave take the 16 tokens of the winning chunk c (support members only), their
// exact keys fl(fl(z_v/T) + g_v), and the first maximum is the token.
constexpr int kDrawThreads = 1024;
__global__ void __launch_bounds__(kDrawThreads) chunk_draw_kernel(SampleArgs a, int32_t* tokens,
                                                                  float* lse, float* logq) {
  const int r = blockIdx.x, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  Partial p{-INFINITY, 0.f, -INFINITY, 0x7fffffff};
  chunk_keys<kDrawThreads, 12>(a, a.L + (long)r * a.ldL, r, 0, a.nch, p);
  for (int off = 32; off >= 1; off >>= 1) {
    Partial o{__shfl_xor(p.m, off), __shfl_xor(p.s, off), __shfl_xor(p.key, off),
              __shfl_xor(p.idx, off)};
    combine(p, o);
  }
  __shared__ Partial red[kDrawThreads / 64];
  if (lane == 0) red[wave] = p;
  __syncthreads();
  if (wave != 0) return;
  p = red[0];
  for (int w = 1; w < kDrawThreads / 64; ++w) combine(p, red[w]);
  const long g = (long)r * a.row_mul + a.row_add;
  const float* z = a.logits + g * a.vocab;
  // the chunk's tokens: lane i < 16 takes token 16 c + i (no chunk: none)
  const int v = p.idx < a.nch ? p.idx * kChunk + lane : a.vocab;
  float key = -INFINITY, zt = -INFINITY;
  if (lane < kChunk && v < a.vocab) {
    const float zv = z[v];
    const bool in = !a.sel || in_support(a.sel[r], zv, v);
    if (in) {
      zt = a.T == 1.f ? zv : zv / a.T;
      uint32_t w[4];
      noise_block(noise_key(a.seed, a.step, 0), (uint32_t)g, (uint32_t)(v >> 2), w);
      key = __fadd_rn(zt, gumbel_from_bits(w[v & 3]));
    }
  }
  int best = key > -INFINITY ? v : 0x7fffffff;
  for (int off = 8; off >= 1; off >>= 1) {   // lanes 0 .. 15: first maximum
    const float k2 = __shfl_xor(key, off);
    const int b2 = __shfl_xor(best, off);
    const float z2 = __shfl_xor(zt, off);
    if (better(k2, b2, key, best)) { key = k2; best = b2; zt = z2; }
  }
  if (lane == 0) {
    const float l = p.m + logf(p.s);
    tokens[g] = best;
    lse[g] = l;
    logq[g] = zt - l;
  }
}

// Eq. 7 for position i of every sequence: z[b][i][v] += (W_c E_c(y))[v] with
// y = y_{i-1}(b), y_0 the anchor (an anchor outside [0, V) reads row 0). A
// workgroup takes kMkV vocabulary entries: their W_c rows reach LDS through
// coalesced 16-byte loads (rows padded by 16 bytes, so the lanes' row reads
// spread over the banks), and the rank vectors of 16 sequences at a time sit
// in LDS as fp32. Its 4 wave-sized groups of threads take 4 of every 16
// sequences each. Each entry's sum runs over the rank index in order with
// separate fp32 multiplies and adds (no fused multiply-add), so the corrected
// logits are a fixed sequence of IEEE operations that the sampler then reads
// like any other logits.
constexpr int kMkRows = 16, kMkThreads = 256, kMkV = 64, kMkPer = kMkRows / (kMkThreads / kMkV);
// 16 bytes as a native vector (arrays of HIP's struct uint4 end up in scratch)
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
template <typename T, int RMAX>   // RMAX: the largest rank the registers hold (64 or 256)
__global__ void __launch_bounds__(kMkThreads) markov_correct_kernel(
    float* logits, int batch, int B, int vocab, int i, const int32_t* anchor,
    const int32_t* tokens, const T* E, const T* W, int rank) {
#pragma clang fp contract(off)   // products and sums rounded separately, as the oracle states
  extern __shared__ __attribute__((aligned(16))) float e_lds[];   // [kMkRows][rank], then W
  constexpr int EPV = 16 / sizeof(T);   // elements per 16-byte piece (8 or 4)
  const int wld = rank + EPV;           // padded W row in LDS (elements)
  T* w_lds = reinterpret_cast<T*>(e_lds + kMkRows * rank);
  const int v0 = blockIdx.x * kMkV;
  const int lv = threadIdx.x & (kMkV - 1), v = v0 + lv;
  const int grp = threadIdx.x / kMkV;   // rows grp * kMkPer .. + kMkPer of each 16
  // Every global load is issued before the first barrier: the W_c rows of the
  // tile, then per chunk of 16 sequences the logits this thread updates and
  // the rank vectors E_c(y) (a token load, then its row); one barrier after
  // they reach LDS. (W_c rows past V repeat the last one.)
  constexpr int kWMax = kMkV * RMAX / EPV / kMkThreads;   // 16-byte pieces per thread
  constexpr int kEMax = kMkRows * RMAX / kMkThreads;      // rank-vector entries per thread
  const int per_row = rank / EPV, wpieces = kMkV * per_row;
  u32x4 wreg[kWMax];
#pragma unroll
  for (int q = 0; q < kWMax; ++q) {
    const int c = threadIdx.x + q * kMkThreads;
    if (c < wpieces) {
      const int r = c / per_row, k = (c - r * per_row) * EPV;
      wreg[q] = *reinterpret_cast<const u32x4*>(W + (long)min(v0 + r, vocab - 1) * rank + k);
    }
  }
  const T* wr = w_lds + lv * wld;
  const float* e0 = e_lds + grp * kMkPer * rank;
  for (int b0 = 0; b0 < batch; b0 += kMkRows) {
    const int nb = min(kMkRows, batch - b0);
    float zold[kMkPer];
#pragma unroll
    for (int r = 0; r < kMkPer; ++r) {
      const int bb = grp * kMkPer + r;
      zold[r] = v < vocab && bb < nb ? logits[((long)(b0 + bb) * B + i) * vocab + v] : 0.f;
    }
    float ereg[kEMax];
#pragma unroll
    for (int q = 0; q < kEMax; ++q) {
      const int idx = threadIdx.x + q * kMkThreads;
      const int bb = idx / rank, k = idx - bb * rank;
      float e = 0.f;
      if (idx < kMkRows * rank && bb < nb) {
        const int b = b0 + bb;
        int y = i == 0 ? anchor[b] : tokens[(long)b * B + i - 1];
        if (y < 0 || y >= vocab) y = 0;
        e = Elem<T>::load(E + (long)y * rank + k);
      }
      ereg[q] = e;
    }
    if (b0 > 0) __syncthreads();   // the previous chunk's LDS reads are done
    if (b0 == 0) {
#pragma unroll
      for (int q = 0; q < kWMax; ++q) {
        const int c = threadIdx.x + q * kMkThreads;
        if (c < wpieces) {
          const int r = c / per_row, k = (c - r * per_row) * EPV;
          *reinterpret_cast<u32x4*>(w_lds + r * wld + k) = wreg[q];
        }
      }
    }
#pragma unroll
    for (int q = 0; q < kEMax; ++q) {
      const int idx = threadIdx.x + q * kMkThreads;
      if (idx < kMkRows * rank) e_lds[idx] = ereg[q];
    }
    __syncthreads();
    float c[kMkPer];
#pragma unroll
    for (int r = 0; r < kMkPer; ++r) c[r] = 0.f;
    for (int k0 = 0; k0 < rank; k0 += 8) {
      float w[8];
#pragma unroll
      for (int h = 0; h < 8 / EPV; ++h) {
        const uint4 raw = *reinterpret_cast<const uint4*>(wr + k0 + h * EPV);
        const T* wv = reinterpret_cast<const T*>(&raw);
#pragma unroll
        for (int e = 0; e < EPV; ++e) w[h * EPV + e] = Elem<T>::load(wv + e);
      }
#pragma unroll
      for (int r = 0; r < kMkPer; ++r) {
        const float4 ea = *reinterpret_cast<const float4*>(e0 + r * rank + k0);
        const float4 eb = *reinterpret_cast<const float4*>(e0 + r * rank + k0 + 4);
        float x = c[r];
        x = x + w[0] * ea.x; x = x + w[1] * ea.y; x = x + w[2] * ea.z; x = x + w[3] * ea.w;
        x = x + w[4] * eb.x; x = x + w[5] * eb.y; x = x + w[6] * eb.z; x = x + w[7] * eb.w;
        c[r] = x;
      }
    }
    if (v < vocab) {
#pragma unroll
      for (int r = 0; r < kMkPer; ++r) {
        const int bb = grp * kMkPer + r;
        if (bb < nb) logits[((long)(b0 + bb) * B + i) * vocab + v] = zold[r] + c[r];
      }
    }
  }
}

// Greedy partial: the first argmax of chunk [sp * chunk, ..) of the row.
__global__ void __launch_bounds__(kThreads) sample_partial_kernel(SampleArgs a) {
  const int sp = blockIdx.x, r = blockIdx.y;
  const int v0 = sp * a.chunk, v1 = min(a.vocab, v0 + a.chunk);
  const float* z = a.logits + ((long)r * a.row_mul + a.row_add) * a.vocab;
  Partial p{-INFINITY, 0.f, -INFINITY, 0x7fffffff};
  argmax_tokens(a, z, v0, v1, p);
  for (int off = 32; off >= 1; off >>= 1) {
    Partial o{__shfl_xor(p.m, off), __shfl_xor(p.s, off), __shfl_xor(p.key, off),
              __shfl_xor(p.idx, off)};
    combine(p, o);
  }
  __shared__ Partial red[kThreads / 64];
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = p;
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < kThreads / 64; ++w) combine(p, red[w]);
    a.part[(long)r * a.splits + sp] = p;
  }
}

// One wave per row (T = 0): the greedy partials in order, the first argmax,
// its logit as lse and log q = 0.
__global__ void __launch_bounds__(64) sample_merge_kernel(SampleArgs a, int32_t* tokens,
                                                          float* lse, float* logq) {
  const int r = blockIdx.x, lane = threadIdx.x;
  Partial p{-INFINITY, 0.f, -INFINITY, 0x7fffffff};
  for (int sp = lane; sp < a.splits; sp += 64) combine(p, a.part[(long)r * a.splits + sp]);
  for (int off = 32; off >= 1; off >>= 1) {
    Partial o{__shfl_xor(p.m, off), __shfl_xor(p.s, off), __shfl_xor(p.key, off),
              __shfl_xor(p.idx, off)};
    combine(p, o);
  }
  if (lane == 0) {
    const long g = (long)r * a.row_mul + a.row_add;
    tokens[g] = p.idx;
    lse[g] = p.key;
    logq[g] = 0.f;
  }
}

__global__ void __launch_bounds__(kThreads) gumbel_fill_kernel(uint64_t seed, uint64_t step,
                                                               uint32_t stream, int rows,
                                                               int vocab, float* out) {
  const int groups = (vocab + kGroup - 1) / kGroup;
  const long total = (long)rows * groups;
  for (long i = blockIdx.x * (long)kThreads + threadIdx.x; i < total;
       i += (long)gridDim.x * kThreads) {
    const int r = (int)(i / groups), c = (int)(i % groups);
    uint32_t bits[kGroup];
    noise_group(seed, step, (uint64_t)r, stream, (uint64_t)c, bits);
#pragma unroll
    for (int k = 0; k < kGroup; ++k) {
      const int v = c * kGroup + k;
      if (v < vocab) out[(long)r * vocab + v] = gumbel_from_bits(bits[k]);
    }
  }
}

}  // namespace

SamplePlan sample_plan(int rows, int vocab) {
  SamplePlan p;
  // T = 0: a chunk of one sweep times the largest power of two that keeps
  // at least 2048 / rows chunks per row (about 2048 workgroups; 4096 measured
  // no faster), one chunk per row from 2048 rows on
  constexpr int sweep = kThreads * kGroup;
  const long target = ((long)vocab * rows + 2047) / 2048;
  int chunk = sweep;
  while (chunk * 2L <= target && chunk < 32 * sweep) chunk *= 2;
  if (rows >= 2048) chunk = (vocab + sweep - 1) / sweep * sweep;
  p.greedy_chunk = chunk;
  p.greedy_splits = (vocab + chunk - 1) / chunk;
  // T > 0: 16-token chunks, their log-masses in rows padded to 4 floats
  p.nch = (vocab + kChunk - 1) / kChunk;
  p.ldL = (p.nch + 3) / 4 * 4;
  return p;
}

int chunk_lse_slice(int rows, int ntok) {
  // tokens per workgroup of chunk_lse_kernel: the range split evenly over
  // max(1, 2048 / rows) workgroups per row (about 2048 in all: one round of
  // resident workgroups), rounded up to whole sweeps of 1024 tokens
  const int per_row = rows >= 2048 ? 1 : 2048 / rows;
  const long even = ((long)ntok + per_row - 1) / per_row;
  return (int)((even + 1023) / 1024 * 1024);
}

size_t sample_part_bytes(int rows, int vocab) {
  const SamplePlan p = sample_plan(rows, vocab);
  const size_t L = ((size_t)rows * p.ldL * sizeof(float) + 255) / 256 * 256;
  return L + (size_t)rows * p.greedy_splits * sizeof(Partial);
}

// Static scratch of ldr_sample_noalloc: the sampler's partials and top-k
// supports for callers that cannot allocate. Host code never passes the
// array's name to a kernel (on the host it is only a stand-in for the symbol);
// it uses the device address hipGetSymbolAddress returns for the current GPU.
static __device__ __align__(256) uint8_t scratch[LDR_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::once_flag g_scratch_once[kMaxDevices];
void* g_scratch_ptr[kMaxDevices];
hipError_t g_scratch_err[kMaxDevices];
}  // namespace

hipError_t noalloc_scratch(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  // once per device, with that device current (the calling thread's)
  std::call_once(g_scratch_once[dev], [dev] {
    void* p = nullptr;
    g_scratch_err[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    g_scratch_ptr[dev] = g_scratch_err[dev] == hipSuccess ? p : nullptr;
  });
  if (g_scratch_err[dev] != hipSuccess) return g_scratch_err[dev];
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

hipError_t launch_topk_select(const float* logits, int rows, int vocab, int k, TopK* sel,
                              hipStream_t st) {
  hipLaunchKernelGGL(topk_select_kernel, dim3(rows), dim3(kSelThreads), 0, st, logits, vocab, k,
                     sel, 1, 0);
  return hipGetLastError();
}

namespace {
// Arguments of the sampler's kernels for `rows` rows, workspace ws (the
// chunk log-masses, then the partials).
SampleArgs sample_args(const float* logits, int rows, int vocab, float temperature,
                       uint64_t seed, uint64_t step, void* ws, int row_mul, int row_add) {
  const SamplePlan pl = sample_plan(rows, vocab);
  SampleArgs a;
  a.logits = logits; a.rows = rows; a.vocab = vocab; a.T = temperature;
  a.seed = seed; a.step = step;
  a.sel = nullptr; a.row_mul = row_mul; a.row_add = row_add;
  a.vec = vocab % 4 == 0 && reinterpret_cast<uintptr_t>(logits) % 16 == 0;
  a.L = static_cast<float*>(ws);
  a.ldL = pl.ldL; a.nch = pl.nch;
  a.part = reinterpret_cast<Partial*>(static_cast<uint8_t*>(ws) +
                                      ((size_t)rows * pl.ldL * sizeof(float) + 255) / 256 * 256);
  a.chunk = pl.greedy_chunk; a.splits = pl.greedy_splits;
  return a;
}

hipError_t chunk_lse(const SampleArgs& a, int v0, int v1, hipStream_t st) {
  if (v0 >= v1) return hipSuccess;
  const int slice = chunk_lse_slice(a.rows, v1 - v0);
  const dim3 grid((unsigned)((v1 - v0 + slice - 1) / slice), (unsigned)a.rows);
  const bool unit = a.T == 1.f, topk = a.sel != nullptr;
#define LDR_CL(U, K, V) \
  hipLaunchKernelGGL((chunk_lse_kernel<U, K, V>), grid, dim3(kThreads), 0, st, a, v0, v1, slice)
  if (a.vec) {
    if (unit) { if (topk) LDR_CL(true, true, true); else LDR_CL(true, false, true); }
    else { if (topk) LDR_CL(false, true, true); else LDR_CL(false, false, true); }
  } else {
    if (unit) { if (topk) LDR_CL(true, true, false); else LDR_CL(true, false, false); }
    else { if (topk) LDR_CL(false, true, false); else LDR_CL(false, false, false); }
  }
#undef LDR_CL
  return hipGetLastError();
}

hipError_t sample_finish(const SampleArgs& a, int32_t* tokens, float* lse, float* logq,
                         hipStream_t st) {
  if (a.T > 0.f) {
    hipLaunchKernelGGL(chunk_draw_kernel, dim3(a.rows), dim3(kDrawThreads), 0, st, a, tokens,
                       lse, logq);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(sample_partial_kernel, dim3(a.splits, a.rows), dim3(kThreads), 0, st, a);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(sample_merge_kernel, dim3(a.rows), dim3(64), 0, st, a, tokens, lse, logq);
  return hipGetLastError();
}
}  // namespace

hipError_t launch_sample(const float* logits, int rows, int vocab, float temperature,
                         int top_k, uint64_t seed, uint64_t step, int32_t* tokens, float* lse,
                         float* logq, void* ws, size_t sel_off, hipStream_t st, int row_mul,
                         int row_add) {
  SampleArgs a = sample_args(logits, rows, vocab, temperature, seed, step, ws, row_mul, row_add);
  if (temperature > 0.f) {
    if (top_k > 0 && top_k < vocab) {  // T = 0 is the argmax either way
      TopK* sel = reinterpret_cast<TopK*>(static_cast<uint8_t*>(ws) + sel_off);
      hipLaunchKernelGGL(topk_select_kernel, dim3(rows), dim3(kSelThreads), 0, st, logits, vocab,
                         top_k, sel, row_mul, row_add);
      const hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
      a.sel = sel;
    }
    const hipError_t e = chunk_lse(a, 0, vocab, st);
    if (e != hipSuccess) return e;
  }
  return sample_finish(a, tokens, lse, logq, st);
}

hipError_t launch_chunk_lse(const float* logits, int rows, int vocab, float temperature, void* ws,
                            int v0, int v1, hipStream_t st) {
  if (temperature <= 0.f || v0 < 0 || v1 > vocab || v0 % kChunk) return hipErrorInvalidValue;
  return chunk_lse(sample_args(logits, rows, vocab, temperature, 0, 0, ws, 1, 0), v0, v1, st);
}

hipError_t launch_sample_finish(const float* logits, int rows, int vocab, float temperature,
                                uint64_t seed, uint64_t step, void* ws, int32_t* tokens,
                                float* lse, float* logq, hipStream_t st) {
  return sample_finish(sample_args(logits, rows, vocab, temperature, seed, step, ws, 1, 0),
                       tokens, lse, logq, st);
}

hipError_t launch_gumbel_fill(uint64_t seed, uint64_t step, int stream, int rows, int vocab,
                              float* out, hipStream_t st) {
  const long groups = (long)rows * ((vocab + kGroup - 1) / kGroup);
  long blocks = (groups + kThreads - 1) / kThreads;
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(gumbel_fill_kernel, dim3((int)(blocks > 0 ? blocks : 1)), dim3(kThreads),
                     0, st, seed, step, (uint32_t)stream, rows, vocab, out);
  return hipGetLastError();
}

hipError_t launch_sample_markov(float* logits, int batch, int B, int vocab, const int32_t* anchor,
                                const void* E, const void* W, int rank, int dtype,
                                float temperature, int top_k, uint64_t seed, uint64_t step,
                                int32_t* tokens, float* lse, float* logq, void* ws,
                                size_t sel_off, hipStream_t st) {
  const int esz = dtype == LDR_BF16 ? 2 : 4;
  const size_t lds = (size_t)kMkRows * rank * sizeof(float) +
                     (size_t)kMkV * (rank + 16 / esz) * esz;
  const dim3 grid((unsigned)((vocab + kMkV - 1) / kMkV));
  for (int i = 0; i < B; ++i) {
#define LDR_MK(T, RM)                                                                        \
  hipLaunchKernelGGL((markov_correct_kernel<T, RM>), grid, dim3(kMkThreads), lds, st, logits, \
                     batch, B, vocab, i, anchor, tokens, static_cast<const T*>(E),            \
                     static_cast<const T*>(W), rank)
    if (dtype == LDR_BF16) {
      if (rank <= 64) LDR_MK(uint16_t, 64); else LDR_MK(uint16_t, 256);
    } else {
      if (rank <= 64) LDR_MK(float, 64); else LDR_MK(float, 256);
    }
#undef LDR_MK
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    e = launch_sample(logits, batch, vocab, temperature, top_k, seed, step, tokens, lse, logq, ws,
                      sel_off, st, B, i);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace ldr
