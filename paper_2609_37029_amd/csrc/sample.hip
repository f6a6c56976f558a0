// Per-position sampling of the factorised proposal (Eq. 8).
//
// Each row of fp32 logits is split into vocabulary chunks. One workgroup per
// (chunk, row) streams its logits once and keeps, per thread, the best
// Gumbel-max key with its token and the running max / sum of exp(z/T) for the
// log-normaliser; a block reduction writes one partial per chunk. Exact keys
// are computed only for tokens that a cheap upper bound cannot rule out. A merge
// kernel combines the chunks of a row in vocabulary order (lower token wins
// ties) and writes the token, lse and log q(y).
//
// The noise is a pure function of (seed, step, row, token): Philox4x32-10
// (Salmon et al., SC 2011; key = the seed, counter (v/4, row, step, stream 0));
// one Philox block serves 4 consecutive tokens, 32 bits each, and a lane takes
// 8 tokens (two blocks) at a time. The uniform u = (2 (bits >> 9) + 1) 2^-24
// is exact, and g = -log(-log u) uses a log made of IEEE fp32 operations only
// (no contraction, correctly rounded division), so the keys fl(fl(z/T) + g)
// are reproducible bit for bit.
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
  int n_a, split, chunk_b;   // chunks below `split` are `chunk` tokens, from it `chunk_b`
  float T; uint64_t seed, step;
  Partial* part;
  const TopK* sel;  // top-k support per row, or null for the full vocabulary
  int row_mul, row_add;  // row r of the launch is logits row (and noise row) r * mul + add
  int chunk0;            // vocabulary chunk of the launch's first workgroup column
  int vec;               // rows start on 16 bytes (V % 4 == 0, aligned logits): 16-byte loads
};

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

// The lane's kGroup = 8 logits of a sweep at v: two 16-byte loads inside the
// chunk [.., v1), else one load per token (-inf past v1).
__device__ inline void load_group(const SampleArgs& a, const float* z, int v, int v1,
                                  float (&zz)[kGroup]) {
  if (a.vec && v + kGroup <= v1) {
    const float4 x = *reinterpret_cast<const float4*>(z + v);
    const float4 y = *reinterpret_cast<const float4*>(z + v + 4);
    zz[0] = x.x; zz[1] = x.y; zz[2] = x.z; zz[3] = x.w;
    zz[4] = y.x; zz[5] = y.y; zz[6] = y.z; zz[7] = y.w;
  } else {
#pragma unroll
    for (int i = 0; i < kGroup; ++i) zz[i] = v + i < v1 ? z[v + i] : -INFINITY;
  }
}

// Greedy steps (T = 0): the first argmax of the chunk, its logits streamed in
// the sampling sweeps' pattern (the next sweep's loads in flight).
__device__ void argmax_tokens(const SampleArgs& a, const float* z, int v0, int v1, Partial& p) {
  constexpr int kSweep = kThreads * kGroup;
  const int lane_off = (int)threadIdx.x * kGroup;
  float znext[kGroup];
  load_group(a, z, v0 + lane_off, v1, znext);
  for (int vb = v0; vb < v1; vb += kSweep) {
    const int v = vb + lane_off;
    float zcur[kGroup];
#pragma unroll
    for (int i = 0; i < kGroup; ++i) zcur[i] = znext[i];
    if (vb + kSweep < v1) load_group(a, z, v + kSweep, v1, znext);
#pragma unroll
    for (int i = 0; i < kGroup; ++i)
      if (v + i < v1 && better(zcur[i], v + i, p.key, p.idx)) { p.key = zcur[i]; p.idx = v + i; }
  }
}

// Temperature sampling. Every lane keeps the lse partial of its tokens and the
// best (key, token) of the candidates it evaluated. A token is a candidate
// unless zt + bound(g) + margin < the lane's best key, which proves that its
// exact key loses; the margin (1e-3 plus 1e-6 relative) covers the rounding of
// the test and of the fixed-sequence log, whose error is below 1e-5 here.
// Candidates go through a per-wave queue in LDS so that the exact key (two
// logs) is computed 64 at a time by full waves.
template <bool UNIT_T, bool TOPK>
__device__ void sample_tokens(const SampleArgs& a, const float* z, int r, int v0, int v1,
                              Partial& p) {
  const TopK sel = TOPK ? a.sel[r] : TopK{0u, 0};
  struct Cand { float zt; uint32_t bits; int v; };
  __shared__ Cand queue[kThreads / 64][128];
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
  auto load8 = [&](int v, float (&zz)[kGroup]) { load_group(a, z, v, v1, zz); };
  constexpr int kSweep = kThreads * kGroup;
  const int lane_off = (int)(threadIdx.x & ~63) * kGroup + lane * kGroup;
  float znext[kGroup];
  load8(v0 + lane_off, znext);
  for (int vb = v0; vb < v1; vb += kSweep) {
    const int v = vb + lane_off;
    float zcur[kGroup];
#pragma unroll
    for (int i = 0; i < kGroup; ++i) zcur[i] = znext[i];
    if (vb + kSweep < v1) load8(v + kSweep, znext);   // the next sweep's logits in flight
    uint32_t bits[kGroup];
    noise_group(a.seed, a.step, (uint64_t)r * a.row_mul + a.row_add, 0, (uint64_t)(v / kGroup),
                bits);
    float zt[kGroup];
    float gm = -INFINITY;
    bool in[kGroup];
#pragma unroll
    for (int i = 0; i < kGroup; ++i) {
      const float zv = zcur[i];
      in[i] = v + i < v1;
      if constexpr (TOPK) {
        const uint32_t u = order_key(zv);
        in[i] = in[i] && (u > sel.tau || (u == sel.tau && v + i <= sel.v_cut));
      }
      zt[i] = in[i] ? (UNIT_T ? zv : zv / a.T) : -INFINITY;  // IEEE division
      gm = fmaxf(gm, zt[i]);
    }
    if (gm > p.m) { p.s *= __expf(p.m - gm); p.m = gm; }
#pragma unroll
    for (int i = 0; i < kGroup; ++i) {
      const bool valid = in[i];
      if (valid) p.s += __expf(zt[i] - p.m);
      const float margin = 1e-3f + 1e-6f * (fabsf(zt[i]) + fabsf(p.key));
      const bool need = valid && !(zt[i] + gumbel_upper(bits[i]) + margin < p.key);
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

__global__ void __launch_bounds__(kThreads) sample_partial_kernel(SampleArgs a) {
  const int sp = blockIdx.x + a.chunk0, r = blockIdx.y;
  const int v0 = sp < a.n_a ? sp * a.chunk : a.split + (sp - a.n_a) * a.chunk_b;
  const int v1 = min(a.vocab, sp < a.n_a ? min(a.split, v0 + a.chunk) : v0 + a.chunk_b);
  const float* z = a.logits + ((long)r * a.row_mul + a.row_add) * a.vocab;
  Partial p{-INFINITY, 0.f, -INFINITY, 0x7fffffff};
  if (a.T == 0.f) {
    argmax_tokens(a, z, v0, v1, p);
  } else if (a.sel) {
    if (a.T == 1.f) sample_tokens<true, true>(a, z, r, v0, v1, p);
    else sample_tokens<false, true>(a, z, r, v0, v1, p);
  } else {
    if (a.T == 1.f) sample_tokens<true, false>(a, z, r, v0, v1, p);
    else sample_tokens<false, false>(a, z, r, v0, v1, p);
  }
  // block reduction of the partials
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

__global__ void __launch_bounds__(64) sample_merge_kernel(SampleArgs a, int32_t* tokens,
                                                          float* lse, float* logq) {
  const int r = blockIdx.x;
  Partial p{-INFINITY, 0.f, -INFINITY, 0x7fffffff};
  for (int sp = threadIdx.x; sp < a.splits; sp += 64) combine(p, a.part[(long)r * a.splits + sp]);
  for (int off = 32; off >= 1; off >>= 1) {
    Partial o{__shfl_xor(p.m, off), __shfl_xor(p.s, off), __shfl_xor(p.key, off),
              __shfl_xor(p.idx, off)};
    combine(p, o);
  }
  if (threadIdx.x == 0) {
    const long g = (long)r * a.row_mul + a.row_add;
    tokens[g] = p.idx;
    if (a.T == 0.f) {
      lse[g] = p.key;
      logq[g] = 0.f;
    } else {
      const float l = p.m + logf(p.s);
      lse[g] = l;
      logq[g] = a.logits[g * a.vocab + p.idx] / a.T - l;
    }
  }
}

__global__ void __launch_bounds__(kThreads) gumbel_fill_kernel(uint64_t seed, uint64_t step,
                                                               int rows, int vocab, float* out) {
  const int groups = (vocab + kGroup - 1) / kGroup;
  const long total = (long)rows * groups;
  for (long i = blockIdx.x * (long)kThreads + threadIdx.x; i < total;
       i += (long)gridDim.x * kThreads) {
    const int r = (int)(i / groups), c = (int)(i % groups);
    uint32_t bits[kGroup];
    noise_group(seed, step, (uint64_t)r, 0, (uint64_t)c, bits);
#pragma unroll
    for (int k = 0; k < kGroup; ++k) {
      const int v = c * kGroup + k;
      if (v < vocab) out[(long)r * vocab + v] = gumbel_from_bits(bits[k]);
    }
  }
}

}  // namespace

SamplePlan sample_plan(int rows, int vocab) {
  // About 2048 workgroups (8 waves per SIMD; 4096 measured no faster): a
  // chunk of one sweep times the largest power of two that keeps at least
  // 2048 / rows chunks per row (from 2048 rows on, one chunk per row).
  // Up to 256 rows and past 65536 tokens, the tokens from the last multiple
  // of 65536 covered by whole 65536-token blocks of the vocabulary head's
  // full rounds (256 column tiles of 256) take one-sweep chunks instead: that
  // region is sampled after the head's last round (ldr_draft_step_sample), by
  // many short workgroups; ldr_sample uses the same plan, so both calls give
  // the same partials and the same results.
  constexpr int sweep = kThreads * kGroup;
  SamplePlan p;
  if (rows >= 2048) {
    p.chunk_a = (vocab + sweep - 1) / sweep * sweep;
    p.n_a = 1; p.split = vocab; p.chunk_b = sweep; p.n_b = 0;
    return p;
  }
  const long target = ((long)vocab * rows + 2047) / 2048;
  int chunk = sweep;
  while (chunk * 2L <= target && chunk < 32 * sweep) chunk *= 2;
  p.chunk_a = chunk;
  p.chunk_b = sweep;
  const int tiles = (vocab + 255) / 256, full = tiles / 256 * 256;
  const int split = full * 256;
  if (rows <= 256 && full > 0 && split < vocab && split % chunk == 0) {
    p.split = split;
    p.n_a = split / chunk;
    p.n_b = (vocab - split + sweep - 1) / sweep;
  } else {
    p.split = vocab;
    p.n_a = (vocab + chunk - 1) / chunk;
    p.n_b = 0;
  }
  return p;
}

int sample_splits(int rows, int vocab) {
  const SamplePlan p = sample_plan(rows, vocab);
  return p.n_a + p.n_b;
}

size_t sample_part_bytes(int rows, int vocab) {
  return (size_t)rows * sample_splits(rows, vocab) * sizeof(Partial);
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

hipError_t launch_sample(const float* logits, int rows, int vocab, float temperature,
                         int top_k, uint64_t seed, uint64_t step, int32_t* tokens, float* lse,
                         float* logq, void* ws, size_t sel_off, hipStream_t st, int row_mul,
                         int row_add) {
  SampleArgs a;
  a.logits = logits; a.rows = rows; a.vocab = vocab; a.T = temperature;
  a.seed = seed; a.step = step; a.part = static_cast<Partial*>(ws);
  a.sel = nullptr; a.row_mul = row_mul; a.row_add = row_add;
  a.vec = vocab % 4 == 0 && reinterpret_cast<uintptr_t>(logits) % 16 == 0;
  if (temperature > 0.f && top_k > 0 && top_k < vocab) {  // T = 0 is the argmax either way
    TopK* sel = reinterpret_cast<TopK*>(static_cast<uint8_t*>(ws) + sel_off);
    hipLaunchKernelGGL(topk_select_kernel, dim3(rows), dim3(kSelThreads), 0, st, logits, vocab,
                       top_k, sel, row_mul, row_add);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    a.sel = sel;
  }
  const SamplePlan pl = sample_plan(rows, vocab);
  a.chunk = pl.chunk_a; a.n_a = pl.n_a; a.split = pl.split; a.chunk_b = pl.chunk_b;
  a.splits = pl.n_a + pl.n_b;
  a.chunk0 = 0;
  hipLaunchKernelGGL(sample_partial_kernel, dim3(a.splits, rows), dim3(kThreads), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(sample_merge_kernel, dim3(rows), dim3(64), 0, st, a, tokens, lse, logq);
  return hipGetLastError();
}

namespace {
SampleArgs full_vocab_args(const float* logits, int rows, int vocab, float temperature,
                           uint64_t seed, uint64_t step, void* ws) {
  SampleArgs a;
  a.logits = logits; a.rows = rows; a.vocab = vocab; a.T = temperature;
  a.seed = seed; a.step = step; a.part = static_cast<Partial*>(ws);
  a.sel = nullptr; a.row_mul = 1; a.row_add = 0;
  a.vec = vocab % 4 == 0 && reinterpret_cast<uintptr_t>(logits) % 16 == 0;
  const SamplePlan pl = sample_plan(rows, vocab);
  a.chunk = pl.chunk_a; a.n_a = pl.n_a; a.split = pl.split; a.chunk_b = pl.chunk_b;
  a.splits = pl.n_a + pl.n_b;
  a.chunk0 = 0;
  return a;
}
}  // namespace

hipError_t launch_sample_partials(const float* logits, int rows, int vocab, float temperature,
                                  uint64_t seed, uint64_t step, void* ws, int c0, int c1,
                                  hipStream_t st) {
  SampleArgs a = full_vocab_args(logits, rows, vocab, temperature, seed, step, ws);
  if (c0 < 0 || c1 > a.splits || c0 >= c1) return hipErrorInvalidValue;
  a.chunk0 = c0;
  hipLaunchKernelGGL(sample_partial_kernel, dim3(c1 - c0, rows), dim3(kThreads), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_sample_merge(const float* logits, int rows, int vocab, float temperature,
                               void* ws, int32_t* tokens, float* lse, float* logq,
                               hipStream_t st) {
  const SampleArgs a = full_vocab_args(logits, rows, vocab, temperature, 0, 0, ws);
  hipLaunchKernelGGL(sample_merge_kernel, dim3(rows), dim3(64), 0, st, a, tokens, lse, logq);
  return hipGetLastError();
}

hipError_t launch_gumbel_fill(uint64_t seed, uint64_t step, int rows, int vocab, float* out,
                              hipStream_t st) {
  const long groups = (long)rows * ((vocab + kGroup - 1) / kGroup);
  long blocks = (groups + kThreads - 1) / kThreads;
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(gumbel_fill_kernel, dim3((int)(blocks > 0 ? blocks : 1)), dim3(kThreads),
                     0, st, seed, step, rows, vocab, out);
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
