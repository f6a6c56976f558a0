// Weight-streaming GEMMs of the drafter: C[M][N] = A[M][K] . W[N][K]^T with
// fp32 accumulation, for the boundary fusion, the QKV / O / gate-up / down
// projections of every layer and the vocabulary head (Sec. 2.3, App. B.1).
//
// With M = batch x B rows (256 at batch 16) these GEMMs stream each weight
// once from HBM and reuse it across all M rows:
//  * a workgroup owns a BM x BN output tile (BM = all M rows up to 256) and a
//    1/splits share of K, with WM x WN waves of MTW x NTW 16x16 MFMA tiles;
//  * both operands reach LDS through coalesced 16-byte loads (8 lanes per
//    128-byte row segment), double-buffered, in 128-byte rows whose 16-byte
//    chunks are XOR-swizzled (lds_chunk) so that both the stores and the
//    16-lane fragment reads of v_mfma_f32_16x16x32_bf16 are conflict-free;
//  * weight loads run WPF steps ahead and activation loads 2 steps ahead in
//    register rings, so HBM latency is covered by several steps of MFMAs;
//  * the loop body has no branches (rows past M or N load a clamped valid
//    row whose results are never stored, prefetches past the last step reload
//    it) and the per-step barrier waits for LDS traffic only, so prefetches
//    stay in flight across it.
// fp32: a plain SIMT tile kernel with the same epilogues.
//
// Epilogues: EPI_STORE writes fp32 (split-K partials); EPI_LOGITS writes the
// fp32 logits; EPI_SWIGLU reads the gate and up rows of w_gate_up interleaved
// in 16-row blocks (each wave's n-tile pairs are matching gate / up columns)
// and writes silu(gate) * up in the activation dtype. The vocabulary head's
// epilogue can also take each row's first argmax (greedy sampling) or form
// the 16-token chunk log-masses of the two-level draw (Eq. 8).
#include "ldr_internal.h"

#include <type_traits>
#include <utility>

namespace ldr {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
// 16 bytes as a native vector (HIP's uint4 is a struct whose copies become
// memcpys that keep arrays of them in scratch).
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int BK = 64;        // K step: one LDS stage, two MFMA k-steps
constexpr int LDK = BK;       // LDS row (elements): 128 B, 16-byte chunks swizzled
// Physical 16-byte chunk of logical chunk c (0..7) in LDS row r: rows r and
// r + 1 sit in opposite halves of the 64 banks, and the 8 row pairs of any 16
// consecutive rows get distinct chunk slots, so both a 16-lane pass of stores
// (two rows of 8 chunks) and of fragment reads (16 rows, one chunk) hit 64
// distinct banks.
__device__ inline int lds_chunk(int r, int c) { return c ^ ((r >> 1) & 7); }

// Interleaved N index of the SwiGLU GEMM -> row of w_gate_up.
__device__ inline int swiglu_row(int c, int mlp) {
  const int blk = c >> 4, out = ((blk >> 1) << 4) | (c & 15);
  return (blk & 1) ? mlp + out : out;
}

__device__ inline float silu(float x) { return x / (1.f + expf(-x)); }
// silu of the bf16 GEMMs, whose result is rounded to bf16: the hardware
// exp2 and reciprocal (about 1 ulp each in fp32) instead of expf and an IEEE
// division, a few VALU operations in place of some thirty.
__device__ inline float silu_bf16(float x) {
  return x * __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(x * -1.44269504088896341f));
}

// One 16 x 16 x 32 MFMA of an activation fragment and a weight fragment.
// TRANS (the SwiGLU GEMMs) takes the weight fragment first, so the
// accumulator tile is transposed: lane l holds columns 4 (l / 16) .. + 3 of
// row l % 16, 4 consecutive outputs of one row. Otherwise lane l holds rows
// 4 (l / 16) .. + 3 of column l % 16. The products and sums are the same
// either way. (The SwiGLU epilogue writes 4 consecutive bf16 at a time; the
// fp32 split-K stores of 4 consecutive columns per lane measured 1 us slower
// for the QKV projection, whose rows lie 24 KB apart, and no faster for the
// others.)
template <bool TRANS>
__device__ __forceinline__ void mma_tile(const bf16x8& a, const bf16x8& w, f32x4& acc) {
  acc = TRANS ? __builtin_amdgcn_mfma_f32_16x16x32_bf16(w, a, acc, 0, 0, 0)
              : __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, w, acc, 0, 0, 0);
}

// acc = A[m0 .., kbeg .. kbeg + nk BK) . W[n0 .., same]^T for one BM x BN tile
// (SWI: W rows in the interleaved gate/up order), through the LDS buffers
// As / Ws of the calling kernel, WPF weight steps in flight in registers.
// nk even (two steps per loop pass).
template <int MTW, int NTW, int WM, int WN, bool SWI, int WPF>
__device__ __forceinline__ void tile_mma(const GemmArgs& a, int n0, int m0, int kbeg, int nk,
                                         uint16_t (&As)[2][WM * MTW * 16 * LDK],
                                         uint16_t (&Ws)[2][WN * NTW * 16 * LDK],
                                         f32x4 (&acc)[MTW][NTW]) {
  constexpr int NTHR = WM * WN * 64, TM = MTW * 16, TN = NTW * 16;
  constexpr int BM = WM * TM, BN = WN * TN;
  constexpr int ACH = BM * (BK / 8), WCH = BN * (BK / 8);   // 16-byte chunks per stage
  constexpr int AL = (ACH + NTHR - 1) / NTHR, WL = (WCH + NTHR - 1) / NTHR;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const uint16_t* A = static_cast<const uint16_t*>(a.A);
  const uint16_t* W = static_cast<const uint16_t*>(a.W);

  // Chunk c of a stage: row c / 8, columns (c % 8) * 8 .. + 8. Threads past
  // the chunk count duplicate an earlier chunk (same value, same place).
  const uint16_t* asrc[AL];
  const uint16_t* wsrc[WL];
  int adst[AL], wdst[WL];
#pragma unroll
  for (int i = 0; i < AL; ++i) {
    const int c = (tid + i * NTHR) % ACH, row = c >> 3, col = (c & 7) * 8;
    asrc[i] = A + (long)min(m0 + row, a.M - 1) * a.lda + kbeg + col;
    adst[i] = row * LDK + lds_chunk(row, c & 7) * 8;
  }
#pragma unroll
  for (int i = 0; i < WL; ++i) {
    const int c = (tid + i * NTHR) % WCH, row = c >> 3, col = (c & 7) * 8;
    const int gn = min(n0 + row, a.N - 1);
    const int wrow = SWI ? swiglu_row(gn, a.mlp) : gn;
    wsrc[i] = W + (long)wrow * a.ldw + kbeg + col;
    wdst[i] = row * LDK + lds_chunk(row, c & 7) * 8;
  }

  // LDS row offsets of this lane's fragment rows (rows are multiples of 16
  // plus lane & 15, so the swizzle depends on lane & 15 alone)
  int ard[MTW], wrd[NTW];
#pragma unroll
  for (int i = 0; i < MTW; ++i) ard[i] = (wm * TM + i * 16 + (lane & 15)) * LDK;
#pragma unroll
  for (int j = 0; j < NTW; ++j) wrd[j] = (wn * TN + j * 16 + (lane & 15)) * LDK;

  // wq[p]: weights of step kt + 1 + p; a0 / a1: activation stages kt + 1 and
  // kt + 2 (roles swap every step). Constant indices only: registers.
  u32x4 wq[WPF][WL];
  u32x4 a0[AL], a1[AL];
#pragma unroll
  for (int i = 0; i < MTW; ++i)
#pragma unroll
    for (int j = 0; j < NTW; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
#define LDR_LOAD(dst, src, kt) dst = *reinterpret_cast<const u32x4*>((src) + (kt) * BK)
#define LDR_STORE(buf_arr, off, v) *reinterpret_cast<u32x4*>(&buf_arr[off]) = (v)
  // One K step: MFMAs on LDS buffer `buf` while stage kt + 2 of A and step
  // kt + 1 + WPF of W are fetched; then stage kt + 1 (A in `cur`, W in wq[0])
  // goes to the other buffer.
#define LDR_STEP(kt, buf, nxt, cur)                                                   \
  {                                                                                   \
    _Pragma("unroll") for (int i = 0; i < AL; ++i)                                    \
        LDR_LOAD(nxt[i], asrc[i], min((kt) + 2, nk - 1));                             \
    _Pragma("unroll") for (int kk = 0; kk < 2; ++kk) {                                \
      bf16x8 bfr[NTW];                                                                \
      _Pragma("unroll") for (int j = 0; j < NTW; ++j) bfr[j] =                        \
          __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(                 \
              &Ws[buf][wrd[j] + lds_chunk(lane & 15, kk * 4 + (lane >> 4)) * 8]));       \
      _Pragma("unroll") for (int i = 0; i < MTW; ++i) {                               \
        const bf16x8 av = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>( \
            &As[buf][ard[i] + lds_chunk(lane & 15, kk * 4 + (lane >> 4)) * 8]));         \
        _Pragma("unroll") for (int j = 0; j < NTW; ++j)                               \
            mma_tile<SWI>(av, bfr[j], acc[i][j]);                                     \
      }                                                                               \
    }                                                                                 \
    _Pragma("unroll") for (int i = 0; i < AL; ++i) LDR_STORE(As[(buf) ^ 1], adst[i], cur[i]); \
    _Pragma("unroll") for (int i = 0; i < WL; ++i) LDR_STORE(Ws[(buf) ^ 1], wdst[i], wq[0][i]); \
    _Pragma("unroll") for (int p = 0; p + 1 < WPF; ++p)                               \
        _Pragma("unroll") for (int i = 0; i < WL; ++i) wq[p][i] = wq[p + 1][i];       \
    _Pragma("unroll") for (int i = 0; i < WL; ++i)                                    \
        LDR_LOAD(wq[WPF - 1][i], wsrc[i], min((kt) + 1 + WPF, nk - 1));               \
    lds_barrier();                                                                    \
  }

  // Prologue: stage 0 into LDS, A stage 1 and W steps 1..WPF in flight.
#pragma unroll
  for (int i = 0; i < AL; ++i) LDR_LOAD(a0[i], asrc[i], 0);
#pragma unroll
  for (int i = 0; i < WL; ++i) LDR_LOAD(wq[0][i], wsrc[i], 0);
#pragma unroll
  for (int i = 0; i < AL; ++i) LDR_STORE(As[0], adst[i], a0[i]);
#pragma unroll
  for (int i = 0; i < WL; ++i) LDR_STORE(Ws[0], wdst[i], wq[0][i]);
#pragma unroll
  for (int p = 0; p < WPF; ++p)
#pragma unroll
    for (int i = 0; i < WL; ++i) LDR_LOAD(wq[p][i], wsrc[i], min(1 + p, nk - 1));
#pragma unroll
  for (int i = 0; i < AL; ++i) LDR_LOAD(a1[i], asrc[i], min(1, nk - 1));
  lds_barrier();
  // Even steps fetch into a0 and park a1; odd steps the other way round.
  // plan_gemm keeps nk even.
  for (int kt = 0; kt < nk; kt += 2) {
    LDR_STEP(kt, 0, a0, a1)
    LDR_STEP(kt + 1, 1, a1, a0)
  }
#undef LDR_STEP
#undef LDR_STORE
#undef LDR_LOAD
}

// Stores one tile's accumulators: EPI_STORE / EPI_LOGITS fp32 (split z at
// z * split_stride), EPI_SWIGLU silu(gate) * up in the activation dtype,
// row-major or in the fragment layout of [M][mlp] (a.out_frag). The fp32
// tiles are in the MFMA's own layout (lane l: rows 4 (l / 16) .. + 3 of column
// l % 16); the SwiGLU tiles are transposed (mma_tile), so a lane writes 4
// consecutive bf16 of one row (8 bytes in either layout). SwiGLU waves whose
// tile lies inside the matrix skip the per-element tests (a wave-uniform
// branch).
template <int MTW, int NTW, int WM, int WN, int EPI>
__device__ __forceinline__ void store_tile(const GemmArgs& a, int n0, int m0, int z,
                                           const f32x4 (&acc)[MTW][NTW]) {
  constexpr int TM = MTW * 16, TN = NTW * 16;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / WN, wn = wave % WN;
  if constexpr (EPI == EPI_STORE || EPI == EPI_LOGITS) {
    const int crow = (lane >> 4) * 4, ccol = lane & 15;
    const int rb = m0 + wm * TM + crow, cb = n0 + wn * TN + ccol;
    float* out = static_cast<float*>(a.out) + (long)z * a.split_stride + (long)rb * a.ldo + cb;
    if (m0 + wm * TM + TM <= a.M && n0 + wn * TN + TN <= a.N) {
      // the wave's tile lies inside the matrix: no per-element tests
#pragma unroll
      for (int i = 0; i < MTW; ++i)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          float* o = out + (long)(i * 16 + v) * a.ldo;
#pragma unroll
          for (int j = 0; j < NTW; ++j) o[j * 16] = acc[i][j][v];
        }
    } else {
#pragma unroll
      for (int i = 0; i < MTW; ++i)
#pragma unroll
        for (int j = 0; j < NTW; ++j)
#pragma unroll
          for (int v = 0; v < 4; ++v)
            if (rb + i * 16 + v < a.M && cb + j * 16 < a.N)
              out[(long)(i * 16 + v) * a.ldo + j * 16] = acc[i][j][v];
    }
  } else {
    const int r0 = m0 + wm * TM + (lane & 15), c4 = (lane >> 4) * 4;
    uint16_t* out = static_cast<uint16_t*>(a.out);
    // n-tiles j (gate) and j + 1 (up) hold the same 16 output columns
    const int ob = (n0 + wn * TN) / 2 + c4;
    const bool full = m0 + wm * TM + TM <= a.M && (n0 + wn * TN + TN) / 2 <= a.mlp &&
                      (a.out_frag || ((a.ldo & 3) == 0 &&
                                      (reinterpret_cast<uintptr_t>(a.out) & 7) == 0));
    auto put = [&](auto full_t) {
      constexpr bool FULL = decltype(full_t)::value;
#pragma unroll
      for (int j = 0; j < NTW; j += 2) {
        const int col = ob + j * 8;
#pragma unroll
        for (int i = 0; i < MTW; ++i) {
          const int row = r0 + i * 16;
          if (!FULL && (row >= a.M || col >= a.mlp)) continue;
          // col % 8 is 0 or 4: the 4 elements stay inside one 8-element run
          // of the fragment layout
          const long off = a.out_frag ? ((long)(row >> 4) * (a.mlp >> 5) + (col >> 5)) * 512 +
                                            ((((col >> 3) & 3) << 4) | (row & 15)) * 8 + (col & 7)
                                      : (long)row * a.ldo + col;
          uint16_t h[4];
#pragma unroll
          for (int v = 0; v < 4; ++v) h[v] = f32_to_bf16(silu_bf16(acc[i][j][v]) * acc[i][j + 1][v]);
          if (FULL) {
            *reinterpret_cast<uint2*>(out + off) =
                uint2{(uint32_t)h[0] | ((uint32_t)h[1] << 16), (uint32_t)h[2] | ((uint32_t)h[3] << 16)};
          } else {
#pragma unroll
            for (int v = 0; v < 4; ++v)
              if (col + v < a.mlp) out[off + v] = h[v];
          }
        }
      }
    };
    if (full) put(std::true_type{});
    else put(std::false_type{});
  }
}

// The tile (x, y) and K split z of this workgroup. Workgroups go to the 8
// XCDs in turn by linear id (id mod 8), and each XCD has its own L2: the
// linear ids are renumbered so that XCD c takes the c-th eighth of the tiles
// in (z, x, y) order. A K split's activation columns are then read into one
// or two XCDs' L2 instead of all eight, and the row tiles of one column tile
// (M above one tile) share their weight columns in one L2.
__device__ __forceinline__ void xcd_tile(int& x, int& y, int& z) {
  const int gx = gridDim.x, gy = gridDim.y;
  const int total = gx * gy * gridDim.z;
  const int lin = blockIdx.x + gx * (blockIdx.y + gy * blockIdx.z);
  const int q = total >> 3, r = total & 7, c = lin & 7, slot = lin >> 3;
  const int l = c < r ? c * (q + 1) + slot : r * (q + 1) + (c - r) * q + slot;
  y = l % gy;
  x = (l / gy) % gx;
  z = l / (gx * gy);
}

// WPF: weight steps in flight (8 measured no faster for the 16-row tiles,
// which only stream weights).
template <int MTW, int NTW, int WM, int WN, int EPI, int WPF = 4>
__global__ void __launch_bounds__(WM * WN * 64, 1) gemm_kernel(GemmArgs a) {
  constexpr int BM = WM * MTW * 16, BN = WN * NTW * 16;
  static_assert(EPI != EPI_SWIGLU || NTW % 2 == 0, "swiglu pairs");
  __shared__ __attribute__((aligned(16))) uint16_t As[2][BM * LDK];
  __shared__ __attribute__((aligned(16))) uint16_t Ws[2][BN * LDK];
  int bx, by, z;
  xcd_tile(bx, by, z);
  const int n0 = bx * BN, m0 = by * BM;
  const int kper = a.K / a.splits, kbeg = z * kper, nk = kper / BK;
  f32x4 acc[MTW][NTW];
  tile_mma<MTW, NTW, WM, WN, EPI == EPI_SWIGLU, WPF>(a, n0, m0, kbeg, nk, As, Ws, acc);
  store_tile<MTW, NTW, WM, WN, EPI>(a, n0, m0, z, acc);
}

// fp32 SIMT tile: 32 x 64 outputs per 256 threads, each 2 rows x 4 columns
// (rows tm + 16r, columns tn + 16c), K step 16.
template <int EPI>
__global__ void __launch_bounds__(256) gemm_f32_kernel(GemmArgs a) {
  constexpr int FBM = 32, FBN = 64, FBK = 16;
  __shared__ float As[FBK][FBM + 1];
  __shared__ float Ws[FBK][FBN + 1];
  const int tid = threadIdx.x, tm = tid >> 4, tn = tid & 15;
  const int n0 = blockIdx.x * FBN, m0 = blockIdx.y * FBM, z = blockIdx.z;
  const int kper = a.K / a.splits, kbeg = z * kper;
  const float* A = static_cast<const float*>(a.A);
  const float* W = static_cast<const float*>(a.W);
  float acc[2][4] = {};
  for (int k0 = kbeg; k0 < kbeg + kper; k0 += FBK) {
    for (int i = tid; i < FBM * FBK; i += 256) {
      const int r = i / FBK, k = i % FBK, gm = m0 + r;
      As[k][r] = (gm < a.M) ? A[(long)gm * a.lda + k0 + k] : 0.f;
    }
    for (int i = tid; i < FBN * FBK; i += 256) {
      const int r = i / FBK, k = i % FBK, gn = n0 + r;
      int wrow = -1;
      if (gn < a.N) wrow = EPI == EPI_SWIGLU ? swiglu_row(gn, a.mlp) : gn;
      Ws[k][r] = wrow >= 0 ? W[(long)wrow * a.ldw + k0 + k] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < FBK; ++k)
#pragma unroll
      for (int r = 0; r < 2; ++r)
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[r][c] += As[k][tm + 16 * r] * Ws[k][tn + 16 * c];
    __syncthreads();
  }
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    const int row = m0 + tm + 16 * r;
    if (row >= a.M) continue;
    if constexpr (EPI == EPI_STORE) {
      float* out = static_cast<float*>(a.out) + (long)z * a.split_stride;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int col = n0 + tn + 16 * c;
        if (col < a.N) out[(long)row * a.ldo + col] = acc[r][c];
      }
    } else {
      float* out = static_cast<float*>(a.out);
#pragma unroll
      for (int c = 0; c < 4; c += 2) {  // columns tn + 16c (gate) and tn + 16(c+1) (up)
        const int col = (n0 + 16 * c) / 2 + tn;
        if (col < a.mlp) out[(long)row * a.ldo + col] = silu(acc[r][c]) * acc[r][c + 1];
      }
    }
  }
}

template <int N> __device__ inline void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}
__device__ inline void wait_lgkmcnt0() { __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (3 << 14)); }
__device__ inline void sched_fence() { __builtin_amdgcn_sched_barrier(0); }
__device__ inline void group_barrier() {
  sched_fence();
  __builtin_amdgcn_s_barrier();
  sched_fence();
}

#define LDR_GP(p) ((__attribute__((address_space(1))) void*)(p))
#define LDR_LP(p) ((__attribute__((address_space(3))) void*)(p))

// ---------------------------------------------------------------------------
// GEMM with the activation rows in the fragment layout.
//
// In the fragment layout of a [M][K] bf16 matrix (rows padded to 16), the
// 16 x 32 block of rows 16 r .. and columns 32 c .. is 1 KB at element
// (r * (K / 32) + c) * 512, its 16-byte chunk l holding row 16 r + (l & 15),
// columns 32 c + (l >> 4) * 8 .. + 8: the A operand of v_mfma_f32_16x16x32_bf16
// for lane l, so a wave loads an A fragment from global memory with one fully
// coalesced 16-byte load per lane. That is, element (m, k) sits at
// ((m >> 4) * (K >> 5) + (k >> 5)) * 512 + ((((k >> 3) & 3) << 4) | (m & 15)) * 8
// + (k & 7). The residual norms, the attention output and the SwiGLU GEMM write
// their rows in that layout for the GEMM that reads them.
//
// A workgroup owns all 256 rows x BN columns of the output and a 1/splits
// share of K, in steps of 64. Eight compute waves own 32 rows each: their A
// fragments go straight to registers, FRA steps ahead (private, so no LDS),
// and they read all BN weight rows of a step from LDS. The same pipeline
// with one compute wave of 16 rows reading row-major activations (ROWA) takes
// the GEMMs of at most 16 rows in place of the staged kernel: those only
// stream their weights, and the DMA streams them faster (the boundary fusion
// at batch 16 35.8 -> 33.5 us; the batch-1 SwiGLU GEMM 53.4 -> 49.8 us). NL loader waves only
// stage the weights by DMA (global_load_lds, 8 rows of 128 bytes per
// instruction, 16-byte chunk c of row r at c ^ (r & 7)) into a ring of NB
// stages, NB - 1 steps ahead. A wave that issued the weight DMA itself
// between its MFMAs ran them at about half their rate; with the DMA in waves
// of its own the compute waves keep most of it.
// Ordering: at step kt every wave waits for its own share of what the step
// needs (a loader: its DMA of stage kt, with the NB - 2 later stages still in
// flight; a compute wave: its A loads of stage kt and its LDS reads of step
// kt - 1), then the step's barrier. After it the loaders refill the buffer of
// stage kt - 1, whose readers are past the barrier, with stage kt + NB - 1,
// and the compute waves read stage kt. Both roles meet the same nk barriers.
template <class F, int... P>
__device__ __forceinline__ void for_phases(F&& f, std::integer_sequence<int, P...>) {
  (f(std::integral_constant<int, P>{}), ...);
}

template <int N> __device__ inline void wait_vm_lgkm0() {
  static_assert(N >= 0 && N < 64, "vmcnt");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (0 << 8) | ((N >> 4) << 14));
}

constexpr int kFragWaves = 8;    // compute waves of the fragment-layout GEMM
constexpr int kFragLoaders = 4;  // its loader waves
constexpr int kFragThreads = 64 * (kFragWaves + kFragLoaders);
constexpr int kRowsThreads = 64 * (1 + kFragLoaders);   // the 16-row variant

// NW compute waves of MTW 16-row tiles each; ROWA: activations row-major
// (row stride lda) instead of the fragment layout.
template <int MTW, int NTW, int EPI, int FRA, int NL, int NB, int NW, bool ROWA>
__device__ __forceinline__ void frag_gemm(const GemmArgs& a) {
  constexpr int WM = NW, WN = 1, TM = MTW * 16, TN = NTW * 16;
  constexpr int BM = WM * TM, BN = WN * TN;
  constexpr int STAGE = BN * 128;             // W bytes per stage (BN rows x 64 k)
  constexpr int GROUPS = BN / 8;              // DMA instructions per stage (8 rows each)
  static_assert(GROUPS % NL == 0, "loaders share the stage evenly");
  constexpr int GPL = GROUPS / NL;            // DMA instructions per loader and stage
  constexpr int AV = MTW * 2;                 // A loads per stage per compute lane
  constexpr int WAIT_W = GPL * (NB - 2);
  constexpr int WAIT_A = AV * (FRA - 1);
  static_assert(WAIT_W < 64 && WAIT_A < 64, "vmcnt range");
  static_assert(NB % FRA == 0, "the unrolled loop cycles both rings");
  static_assert(EPI != EPI_SWIGLU || NTW % 2 == 0, "swiglu pairs");
  __shared__ __attribute__((aligned(1024))) uint8_t Wsm[NB * STAGE];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int bx, by, z;
  xcd_tile(bx, by, z);
  const int n0 = bx * BN, m0 = by * BM;
  const int kper = a.K / a.splits, kbeg = z * kper, nk = kper / BK;
  if (wave >= NW) {
    // loader l: groups l * GPL .. + GPL of every stage; lane -> row g * 8 +
    // lane / 8, physical chunk lane % 8 <- logical chunk (lane % 8) ^ (row & 7);
    // weight rows past N repeat the last one (their columns are not stored)
    const int l = wave - NW;
    const uint16_t* W = static_cast<const uint16_t*>(a.W);
    const uint16_t* wsrc[GPL];
    int wdst[GPL];
#pragma unroll
    for (int q = 0; q < GPL; ++q) {
      const int g = l * GPL + q;
      const int r = g * 8 + (lane >> 3);
      const int c = (lane & 7) ^ (r & 7);
      const int gn = min(n0 + r, a.N - 1);
      const int wrow = EPI == EPI_SWIGLU ? swiglu_row(gn, a.mlp) : gn;
      wsrc[q] = W + (long)wrow * a.ldw + kbeg + c * 8;
      wdst[q] = g * 1024;
    }
    auto issue_w = [&](int buf, int stage) {   // stages past the end reload the last one
      const int off = min(stage, nk - 1) * BK;
      uint8_t* dst = Wsm + buf * STAGE;
#pragma unroll
      for (int q = 0; q < GPL; ++q)
        __builtin_amdgcn_global_load_lds(LDR_GP(wsrc[q] + off), LDR_LP(dst + wdst[q]), 16, 0, 0);
    };
#pragma unroll
    for (int st = 0; st < NB - 1; ++st) issue_w(st, st);
    int buf = NB - 1;
    for (int kt = 0; kt < nk; ++kt) {
      wait_vmcnt<WAIT_W>();
      group_barrier();
      issue_w(buf, kt + NB - 1);
      buf = buf == NB - 1 ? 0 : buf + 1;
    }
    wait_vmcnt<0>();   // no DMA outlives the workgroup
    return;
  }
  const int wm = wave;
  const uint16_t* A = static_cast<const uint16_t*>(a.A);
  // A fragments of m-tile i and k half kk of a step: in the fragment layout
  // one 1 KB block each (row blocks past the padded row count repeat the
  // last one); row-major, lane l reads row l % 16 (rows past M repeat the
  // last one), 8 columns from (l / 16) * 8. Those rows are never stored.
  const uint16_t* asrc[MTW];
  if constexpr (ROWA) {
#pragma unroll
    for (int i = 0; i < MTW; ++i) {
      const int r = min(m0 + wm * TM + i * 16 + (lane & 15), a.M - 1);
      asrc[i] = A + (long)r * a.lda + kbeg + (lane >> 4) * 8;
    }
  } else {
    const int mpad = (a.M + 15) & ~15;
#pragma unroll
    for (int i = 0; i < MTW; ++i) {
      const int rg = min(m0 + wm * TM + i * 16, mpad - 16) >> 4;
      asrc[i] = A + ((long)rg * (a.K >> 5) + (kbeg >> 5)) * 512 + lane * 8;
    }
  }
  constexpr int KKA = ROWA ? 32 : 512;       // elements between the two k halves
  constexpr long STA = ROWA ? BK : 1024;     // elements between steps
  u32x4 aq[FRA][MTW][2];
  auto load_a = [&](u32x4 (&dst)[MTW][2], int stage) {   // past the end: the last stage again
    const long off = (long)min(stage, nk - 1) * STA;
#pragma unroll
    for (int i = 0; i < MTW; ++i)
#pragma unroll
      for (int kk = 0; kk < 2; ++kk)
        dst[i][kk] = *reinterpret_cast<const u32x4*>(asrc[i] + off + kk * KKA);
  };
  // W fragment offsets in a stage: row j * 16 + lane % 16, logical chunk
  // kk * 4 + lane / 16
  int woff[NTW][2];
#pragma unroll
  for (int j = 0; j < NTW; ++j)
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const int r = j * 16 + (lane & 15);
      woff[j][kk] = r * 128 + (((kk * 4 + (lane >> 4)) ^ (r & 7)) * 16);
    }
  f32x4 acc[MTW][NTW];
#pragma unroll
  for (int i = 0; i < MTW; ++i)
#pragma unroll
    for (int j = 0; j < NTW; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int st = 0; st < FRA; ++st) load_a(aq[st], st);
  // step kt in phase p = kt mod NB: W stage kt in buffer p, A stage kt in
  // register slot p mod FRA, refilled with stage kt + FRA after the MFMAs
  auto step = [&](int kt, auto pc) {
    constexpr int p = decltype(pc)::value;
    sched_fence();
    wait_vm_lgkm0<WAIT_A>();
    __builtin_amdgcn_s_barrier();
    sched_fence();
    const uint8_t* cur = Wsm + p * STAGE;
    bf16x8 bfr[2][NTW];
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int j = 0; j < NTW; ++j)
        bfr[kk][j] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(cur + woff[j][kk]));
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int i = 0; i < MTW; ++i)
#pragma unroll
        for (int j = 0; j < NTW; ++j)
          mma_tile<EPI == EPI_SWIGLU>(__builtin_bit_cast(bf16x8, aq[p % FRA][i][kk]), bfr[kk][j],
                                      acc[i][j]);
    load_a(aq[p % FRA], kt + FRA);
    sched_fence();
  };
  const int full = nk / NB * NB;
  int kt = 0;
  for (; kt < full; kt += NB)
    for_phases([&](auto pc) { step(kt + decltype(pc)::value, pc); },
               std::make_integer_sequence<int, NB>{});
  const int rem = nk - full;   // uniform: every wave takes the same steps
  for_phases([&](auto pc) { if (decltype(pc)::value < rem) step(kt + decltype(pc)::value, pc); },
             std::make_integer_sequence<int, NB - 1>{});
  wait_vm_lgkm0<0>();
  store_tile<MTW, NTW, WM, WN, EPI>(a, n0, m0, z, acc);
}

template <int MTW, int NTW, int EPI, int FRA, int NL, int NB>
__global__ void __launch_bounds__(64 * (kFragWaves + NL), 1) gemm_frag_kernel(GemmArgs a) {
  frag_gemm<MTW, NTW, EPI, FRA, NL, NB, kFragWaves, false>(a);
}

// M <= 16, row-major activations: one compute wave and the loader waves.
template <int NTW, int EPI>
__global__ void __launch_bounds__(kRowsThreads, 1) gemm_rows16_kernel(GemmArgs a) {
  frag_gemm<1, NTW, EPI, 2, kFragLoaders, 6, 1, true>(a);
}

// ---------------------------------------------------------------------------
// GEMM on tiled operands (the vocabulary head).
//
// The activation rows arrive tiled in blocks of TR = 256 rows by TK = 32
// columns, block (r / TR, k / TK) at ((r / TR) * (K / TK) + k / TK) * TR * TK,
// its rows contiguous (TK elements each); the weight [N][K] in column blocks:
// element (n, k) at (k / TK) * R * TK + n * TK + k % TK, R = N rounded up to
// 256 (the layout ldr_tile_matrix writes). One K block of any run of weight
// rows, and of one activation row tile, is then consecutive memory that HBM
// streams at full rate; the same rows read in row-major order are 64-byte
// pieces 8 KB apart, which it serves at about half.
//
// A workgroup of 8 waves owns a 256 x HB output tile, HB = 304 = 19 x 16
// columns: the vocabulary of 151936 then makes 500 tiles, under two rounds
// over the 256 CUs (256-column tiles would make 594: a third round of 82
// tiles that runs nearly as long as a full one, at one CU's streaming rate).
// The waves compute 128 x 80 each (8 x 5 MFMA tiles), so the tile computes
// HW = 320 columns; the last 16 belong to the next tile: their weight rows
// are not staged and their columns are dropped.
// Waves 0-3 and 4-7 form two groups that share the four SIMDs pairwise and take
// turns, one barrier apart: while one group issues its 40 MFMAs for the current
// K block, the other reads its fragments of that block from LDS and starts the
// DMA (global_load_lds) of its part of the block D steps ahead: group 0 the
// 256 A rows (16 KB), group 1 the 304 W rows (19 KB). Each SIMD's matrix unit
// is thus fed by one wave or the other most of the time. Stages of 576 rows x
// 64 B live in NB = 4 LDS buffers; the 16-byte chunk c of stage row r sits at
// chunk c ^ ((r >> 2) & 3), so the 16 lanes of a fragment read hit 64 distinct
// banks.
//
// Ordering (t = K block, barriers numbered from the start of the loop):
//  * group 0 reads block t between barriers 2t and 2t + 1, group 1 between
//    2t + 1 and 2t + 2; each waits for its own LDS reads before the barrier that
//    ends its memory phase, so a buffer's last reader is done two barriers
//    before the DMA that refills it (D = NB - 1) is issued;
//  * every wave waits for its own DMA of block t + 1 (vmcnt) before barrier
//    2t + 2, after which block t + 1 is whole in LDS for both groups.
constexpr int TR = 256, TK = 32;
constexpr long TBLK = (long)TR * TK;
constexpr int HB = 304, HW = 320;

__device__ inline int tile_swz(int r) { return (r >> 2) & 3; }
// The 16 rows of wave wq's DMA issue q past the tile's HB columns.
__device__ inline bool lr_overlap(int wq, int q) { return wq * 80 + q * 16 >= HB; }

// Greedy partial of the fused head: the largest logit of a column range and
// its first token.
struct HeadPart { float key; int idx; };

__device__ inline void head_combine(HeadPart& a, const HeadPart& b) {
  if (b.key > a.key || (b.key == a.key && b.idx < a.idx)) a = b;
}

// Epilogues of the vocabulary head: logits only; the greedy partials (logits
// optional); the logits and the chunk log-masses at T > 0 (T = 1 without the
// division).
constexpr int kHeadLogits = 0, kHeadArgmax = 1, kHeadChunks = 2, kHeadChunksUnitT = 3;

template <int HS>
__global__ void __launch_bounds__(512, 1) gemm_tiled_kernel(GemmArgs a, HeadSampleArgs hs) {
  constexpr int NB = 4, D = NB - 1;
  constexpr int STAGE = (TR + HW) * TK * 2;   // bytes: A rows 0..255, W rows 256..575
  constexpr int MT = 8, NT = 5;               // 16 x 16 MFMA tiles per wave: 128 x 80
  constexpr int QA = TR / 64, QW = HW / 64;   // DMA issues per lane: 4 (A), 5 (W)
  __shared__ __attribute__((aligned(1024))) uint8_t S0[STAGE];
  __shared__ __attribute__((aligned(1024))) uint8_t S1[STAGE];
  __shared__ __attribute__((aligned(1024))) uint8_t S2[STAGE];
  __shared__ __attribute__((aligned(1024))) uint8_t S3[STAGE];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int grp = wave >> 2, wq = wave & 3;
  const int wm = grp, wn = wq;   // output rows wm * 128 .., columns wn * 80 ..
  const int nkb = a.K / TK;
  int ct, rt, z_;
  xcd_tile(ct, rt, z_);   // column tile, row tile: the row tiles of a column tile share its
                          // weight columns in one L2
  const int n0 = ct * HB;
  // DMA: wave wq of group 0 moves A rows wq * 64 + q * 16 + lane / 4, of group 1
  // W rows wq * 80 + q * 16 + lane / 4 (4 lanes per 64-byte row, lane & 3 = the
  // destination chunk); W rows past the padded matrix read its last row.
  const uint16_t* src[QW];
  int dst[QW];
  long kstride;
  if (grp == 0) {
    const uint16_t* tile = static_cast<const uint16_t*>(a.A) + (long)rt * nkb * TBLK;
#pragma unroll
    for (int q = 0; q < QW; ++q) {
      const int r = wq * 64 + (q < QA ? q : 0) * 16 + (lane >> 2);
      src[q] = tile + r * TK + (((lane & 3) ^ tile_swz(r)) * 8);
      dst[q] = (wq * 64 + (q < QA ? q : 0) * 16) * 64;
    }
    kstride = TBLK;
  } else {
    // The last 16 of the 320 rows belong to the next tile; their output
    // columns are dropped. Their DMA (wave 3, q = 4) re-reads the 16 rows
    // before them, which the same wave has just requested (a cache hit, with
    // the same chunk swizzle), instead of fetching 16 more rows from memory:
    // every wave still issues QW DMAs per block.
    const long R = a.ldw;   // padded weight rows of one column block
#pragma unroll
    for (int q = 0; q < QW; ++q) {
      const int lr = wq * 80 + q * 16 + (lane >> 2) - (lr_overlap(wq, q) ? 16 : 0);
      const long gr = min((long)n0 + lr, R - 1);
      src[q] = static_cast<const uint16_t*>(a.W) + gr * TK +
               (((lane & 3) ^ tile_swz(TR + lr)) * 8);
      dst[q] = (TR + wq * 80 + q * 16) * 64;
    }
    kstride = R * TK;
  }
  // Blocks past the end reload the last one (never read).
  auto issue_a = [&](uint8_t* buf, int t) {
    const long off = (long)min(t, nkb - 1) * kstride;
#pragma unroll
    for (int q = 0; q < QA; ++q)
      __builtin_amdgcn_global_load_lds(LDR_GP(src[q] + off), LDR_LP(buf + dst[q]), 16, 0, 0);
  };
  auto issue_w = [&](uint8_t* buf, int t) {
    const long off = (long)min(t, nkb - 1) * kstride;
#pragma unroll
    for (int q = 0; q < QW; ++q)
      __builtin_amdgcn_global_load_lds(LDR_GP(src[q] + off), LDR_LP(buf + dst[q]), 16, 0, 0);
  };
  int aoff[MT], woff[NT];
#pragma unroll
  for (int i = 0; i < MT; ++i) {
    const int r = wm * 128 + i * 16 + (lane & 15);
    aoff[i] = r * 64 + (((lane >> 4) ^ tile_swz(r)) * 16);
  }
#pragma unroll
  for (int j = 0; j < NT; ++j) {
    const int r = TR + wn * 80 + j * 16 + (lane & 15);
    woff[j] = r * 64 + (((lane >> 4) ^ tile_swz(r)) * 16);
  }
  f32x4 acc[MT][NT];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NT; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  bf16x8 af[MT], bfr[NT];

#define LDR_MEM(t, cur, nxt, ISSUE)                                                            \
  {                                                                                            \
    sched_fence();                                                                             \
    _Pragma("unroll") for (int i = 0; i < MT; ++i) af[i] =                                     \
        __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(cur + aoff[i]));            \
    _Pragma("unroll") for (int j = 0; j < NT; ++j) bfr[j] =                                    \
        __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(cur + woff[j]));            \
    ISSUE(nxt, (t) + D);                                                                       \
    sched_fence();                                                                             \
    wait_lgkmcnt0();                                                                           \
  }
#define LDR_MMA()                                                                              \
  {                                                                                            \
    sched_fence();                                                                             \
    __builtin_amdgcn_s_setprio(1);                                                             \
    _Pragma("unroll") for (int i = 0; i < MT; ++i)                                             \
      _Pragma("unroll") for (int j = 0; j < NT; ++j) acc[i][j] =                               \
          __builtin_amdgcn_mfma_f32_16x16x32_bf16(bfr[j], af[i], acc[i][j], 0, 0, 0);          \
    __builtin_amdgcn_s_setprio(0);                                                             \
    sched_fence();                                                                             \
  }
#define LDR_G0(t, cur, nxt) { LDR_MEM(t, cur, nxt, issue_a) group_barrier(); LDR_MMA() wait_vmcnt<QA * (D - 1)>(); group_barrier(); }
#define LDR_G1(t, cur, nxt) { LDR_MEM(t, cur, nxt, issue_w) wait_vmcnt<QW * (D - 1)>(); group_barrier(); LDR_MMA() group_barrier(); }
  if (grp == 0) { issue_a(S0, 0); issue_a(S1, 1); issue_a(S2, 2); }
  else { issue_w(S0, 0); issue_w(S1, 1); issue_w(S2, 2); }
  wait_vmcnt<0>();
  group_barrier();
  if (grp == 0) {
    for (int t = 0; t < nkb; t += NB) {
      LDR_G0(t, S0, S3) LDR_G0(t + 1, S1, S0) LDR_G0(t + 2, S2, S1) LDR_G0(t + 3, S3, S2)
    }
    group_barrier();   // pairs with group 1's offset barrier
  } else {
    group_barrier();   // offset: group 1 starts one barrier later
    for (int t = 0; t < nkb; t += NB) {
      LDR_G1(t, S0, S3) LDR_G1(t + 1, S1, S0) LDR_G1(t + 2, S2, S1) LDR_G1(t + 3, S3, S2)
    }
  }
#undef LDR_G1
#undef LDR_G0
#undef LDR_MMA
#undef LDR_MEM
  wait_vmcnt<0>();   // no DMA outlives the workgroup
  // The MFMAs take the weight fragments as their first operand, so each
  // 16 x 16 accumulator tile is (token, row): lane l holds 4 consecutive
  // tokens g * 4 .. + 3 (g = l / 16) of row l % 16, one float4 of logits, and
  // the 4 lanes g = 0 .. 3 of a row hold one 16-token chunk.
  const int g = lane >> 4, rl = lane & 15;
  const int r0 = rt * TR + wm * 128, c0 = n0 + wn * 80;
  const int cend = min(a.N, n0 + HB);   // the tile's own columns
  // Most waves hold no token past the vocabulary and write rows that start
  // on 16 bytes: their epilogues skip the per-token tests (wave-uniform).
  const bool full = c0 + NT * 16 <= a.N && (a.ldo & 3) == 0;
  if (HS != kHeadArgmax || hs.store_logits) {
    float* out = static_cast<float*>(a.out);
    auto store = [&](auto full_t) {
      constexpr bool FULL = decltype(full_t)::value;
#pragma unroll
      for (int i = 0; i < MT; ++i) {
        const int row = r0 + i * 16 + rl;
        if (row >= a.M) continue;
        float* orow = out + (long)row * a.ldo + c0 + g * 4;
#pragma unroll
        for (int j = 0; j < NT; ++j) {
          const int col = c0 + j * 16 + g * 4;
          float* o = orow + j * 16;
          if (FULL) {
            if (c0 + j * 16 < cend) *reinterpret_cast<f32x4*>(o) = acc[i][j];
          } else {
#pragma unroll
            for (int v = 0; v < 4; ++v)
              if (col + v < cend) o[v] = acc[i][j][v];
          }
        }
      }
    };
    if (full) store(std::true_type{});
    else store(std::false_type{});
  }
  // Lane exchanges across the row groups: xor 16 (a swizzle inside each half
  // wave) and xor 32 (a permute).
  auto x16 = [](float x) {
    return __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, x),
                                                                 0x401F));
  };
  const int perm32 = (lane ^ 32) << 2;
  auto x32 = [perm32](float x) {
    return __builtin_bit_cast(float,
                              __builtin_amdgcn_ds_bpermute(perm32, __builtin_bit_cast(int, x)));
  };
  if constexpr (HS == kHeadChunks || HS == kHeadChunksUnitT) {
    // Chunk log-masses (the first level of the two-level draw of Eq. 8 at
    // T > 0): each lane's max and sum of exp(z/T - max) over its 4 tokens,
    // (t0 + t1) + (t2 + t3), then over the chunk's 4 lanes (xor 16, then
    // xor 32) -- the order and operations of the log-mass pass over stored
    // logits, so L_c has the same bits. Tokens past the vocabulary count as
    // -inf; chunks past the tile's own columns belong to the next tile and
    // are not written. Lane group g keeps chunk g (group 0 also chunk 4).
    const float T = hs.T;
    auto chunks = [&](auto full_t) {
      constexpr bool FULL = decltype(full_t)::value;
      // IP row blocks of NT chunks side by side, one phase at a time, so that
      // each lane exchange waits once for all of them
      constexpr int IP = 2;
#pragma unroll
      for (int i0 = 0; i0 < MT; i0 += IP) {
        float zt[IP][NT][4], m[IP][NT], sum[IP][NT], o16[IP][NT], o32[IP][NT];
#pragma unroll
        for (int ii = 0; ii < IP; ++ii)
#pragma unroll
          for (int j = 0; j < NT; ++j) {
            const int col = c0 + j * 16 + g * 4;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
              const float x = acc[i0 + ii][j][v];
              zt[ii][j][v] = FULL || col + v < a.N ? (HS == kHeadChunksUnitT ? x : x / T)
                                                   : -INFINITY;
            }
            m[ii][j] = fmaxf(fmaxf(zt[ii][j][0], zt[ii][j][1]), fmaxf(zt[ii][j][2], zt[ii][j][3]));
          }
#pragma unroll
        for (int ii = 0; ii < IP; ++ii)
#pragma unroll
          for (int j = 0; j < NT; ++j) o16[ii][j] = x16(m[ii][j]);
#pragma unroll
        for (int ii = 0; ii < IP; ++ii)
#pragma unroll
          for (int j = 0; j < NT; ++j) m[ii][j] = fmaxf(m[ii][j], o16[ii][j]);
#pragma unroll
        for (int ii = 0; ii < IP; ++ii)
#pragma unroll
          for (int j = 0; j < NT; ++j) o32[ii][j] = x32(m[ii][j]);
#pragma unroll
        for (int ii = 0; ii < IP; ++ii)
#pragma unroll
          for (int j = 0; j < NT; ++j) {
            m[ii][j] = fmaxf(m[ii][j], o32[ii][j]);
            float e[4];
#pragma unroll
            for (int v = 0; v < 4; ++v) e[v] = chunk_term(zt[ii][j][v], m[ii][j]);
            sum[ii][j] = (e[0] + e[1]) + (e[2] + e[3]);
          }
#pragma unroll
        for (int ii = 0; ii < IP; ++ii)
#pragma unroll
          for (int j = 0; j < NT; ++j) o16[ii][j] = x16(sum[ii][j]);
#pragma unroll
        for (int ii = 0; ii < IP; ++ii)
#pragma unroll
          for (int j = 0; j < NT; ++j) sum[ii][j] += o16[ii][j];
#pragma unroll
        for (int ii = 0; ii < IP; ++ii)
#pragma unroll
          for (int j = 0; j < NT; ++j) o32[ii][j] = x32(sum[ii][j]);
#pragma unroll
        for (int ii = 0; ii < IP; ++ii) {
          float keep = 0.f, keep4 = 0.f;
#pragma unroll
          for (int j = 0; j < NT; ++j) {
            sum[ii][j] += o32[ii][j];
            const float L = chunk_log_mass(m[ii][j], sum[ii][j]);
            if (j == 4) keep4 = L;
            else keep = g == j ? L : keep;
          }
          const int row = r0 + (i0 + ii) * 16 + rl;
          if (row < a.M) {
            float* Lr = hs.L + (long)row * hs.ldL + c0 / 16;
            if (c0 + g * 16 < cend) Lr[g] = keep;
            if (NT > 4 && g == 0 && c0 + 64 < cend) Lr[4] = keep4;
          }
        }
      }
    };
    if (full) chunks(std::true_type{});
    else chunks(std::false_type{});
  }
  if constexpr (HS == kHeadArgmax) {
    // Greedy epilogue (Eq. 8 at T = 0: the first argmax of each row). Per row
    // of the tile: each lane's best of its 20 tokens, the 4 lanes of the row
    // (its 80 columns of this wave) by lane exchanges, the 4 waves of the row
    // through LDS, one partial per (row, column tile).
    __shared__ HeadPart tab[TR][4];
    HeadPart* parts = static_cast<HeadPart*>(hs.parts);
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      HeadPart p{-INFINITY, 0x7fffffff};
#pragma unroll
      for (int j = 0; j < NT; ++j)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int col = c0 + j * 16 + g * 4 + v;
          if (col < cend) head_combine(p, HeadPart{acc[i][j][v], col});
        }
      HeadPart o;
      o.key = x16(p.key);
      o.idx = __builtin_amdgcn_ds_swizzle(p.idx, 0x401F);
      head_combine(p, o);
      o.key = x32(p.key);
      o.idx = __builtin_amdgcn_ds_bpermute(perm32, p.idx);
      head_combine(p, o);
      if (g == 0) tab[wm * 128 + i * 16 + rl][wn] = p;
    }
    __syncthreads();
    if (tid < TR) {
      const int row = rt * TR + tid;
      HeadPart p = tab[tid][0];
#pragma unroll
      for (int q = 1; q < 4; ++q) head_combine(p, tab[tid][q]);
      if (row < a.M) parts[(long)row * hs.nparts + ct] = p;
    }
  }
}

// One wave per row: the column tiles' partials, then the first argmax, its
// logit as lse and log q = 0, as the separate sampler reports them at T = 0.
__global__ void __launch_bounds__(64) head_argmax_merge_kernel(const HeadPart* parts, int nparts,
                                                               int32_t* tokens, float* lse,
                                                               float* logq) {
  const int r = blockIdx.x;
  HeadPart p{-INFINITY, 0x7fffffff};
  for (int s = threadIdx.x; s < nparts; s += 64) head_combine(p, parts[(long)r * nparts + s]);
  for (int off = 32; off >= 1; off >>= 1)
    head_combine(p, HeadPart{__shfl_xor(p.key, off), __shfl_xor(p.idx, off)});
  if (threadIdx.x == 0) {
    tokens[r] = p.idx;
    lse[r] = p.key;
    logq[r] = 0.f;
  }
}

// Column-block copy of a row-major [rows][cols] 2-byte matrix (the weight
// layout of the vocabulary head): one thread per 16-byte chunk of the
// destination, whose column block kb holds R = rows rounded up to 256 rows
// of TK elements; padding rows are zero.
__global__ void __launch_bounds__(256) tile_matrix_kernel(const uint16_t* src, long ld, int rows,
                                                          long R, uint16_t* dst, long chunks) {
  for (long e = (long)blockIdx.x * blockDim.x + threadIdx.x; e < chunks;
       e += (long)gridDim.x * blockDim.x) {
    const long kb = e / (R * (TK / 8));
    const long in = e % (R * (TK / 8));
    const long row = in / (TK / 8);
    const int col = (int)(kb * TK + (in % (TK / 8)) * 8);
    u32x4 v = u32x4{0u, 0u, 0u, 0u};
    if (row < rows) v = *reinterpret_cast<const u32x4*>(src + row * ld + col);
    *reinterpret_cast<u32x4*>(dst + e * 8) = v;
  }
}

// Tile configurations (cfg): 0: BM 16 (M <= 16) with 4 waves along N (BN 128);
// 1: BM 32, 2: BM 64, with 8 waves along N (BN 256); 3: BM 256 with 4 x 2 waves
// of 64 x 64 (BN 128);
// 4: BM 256 with 8 x 1 waves of 32 x 96 (BN 96), for the SwiGLU GEMM, whose
// 2 x 12288 columns at the Qwen3-8B shape make exactly 256 tiles (one per CU);
// 5: BM 256 with 4 x 2 waves of 64 x 32 (BN 64), in place of cfg 3 when cfg 3
// would split K eight ways into pieces of at most 512: as fast there (the O
// projection) with half the split-K partials for the next kernel to read;
// 9: BM 16 with 3 waves along N (BN 96), in place of cfg 0 where 96-column
// tiles fill the CUs better;
// 10, 11: gemm_rows16_kernel, cfg 0 and 9 (BM 16, BN 128 or 96) with the
// weights streamed by loader waves, where each split's K range is a multiple
// of 64;
// 6, 7, 8: gemm_frag_kernel, BM 256 with 8 compute waves of 32 x 96 (BN 96),
// 32 x 128 (BN 128) or 32 x 64 (BN 64) and 4 loader waves, activation rows in
// the fragment layout: the GEMMs above 64 rows whose input is written in that
// layout (the SwiGLU GEMM in place of cfg 4 or 3; the QKV, O and down
// projections).
template <int EPI>
hipError_t launch_cfg(int cfg, dim3 grid, const GemmArgs& a, hipStream_t st) {
  switch (cfg) {
    case 0: hipLaunchKernelGGL((gemm_kernel<1, 2, 1, 4, EPI>), grid, dim3(256), 0, st, a); break;
    case 1: hipLaunchKernelGGL((gemm_kernel<2, 2, 1, 8, EPI>), grid, dim3(512), 0, st, a); break;
    case 2: hipLaunchKernelGGL((gemm_kernel<4, 2, 1, 8, EPI>), grid, dim3(512), 0, st, a); break;
    case 4: hipLaunchKernelGGL((gemm_kernel<2, 6, 8, 1, EPI>), grid, dim3(512), 0, st, a); break;
    case 5: hipLaunchKernelGGL((gemm_kernel<4, 2, 4, 2, EPI>), grid, dim3(512), 0, st, a); break;
    case 6:
      hipLaunchKernelGGL((gemm_frag_kernel<2, 6, EPI, 2, kFragLoaders, 6>), grid,
                         dim3(kFragThreads), 0, st, a);
      break;
    case 7:
      hipLaunchKernelGGL((gemm_frag_kernel<2, 8, EPI, 2, kFragLoaders, 6>), grid,
                         dim3(kFragThreads), 0, st, a);
      break;
    case 8:
      hipLaunchKernelGGL((gemm_frag_kernel<2, 4, EPI, 2, kFragLoaders, 6>), grid,
                         dim3(kFragThreads), 0, st, a);
      break;
    case 9: hipLaunchKernelGGL((gemm_kernel<1, 2, 1, 3, EPI>), grid, dim3(192), 0, st, a); break;
    case 10:
      hipLaunchKernelGGL((gemm_rows16_kernel<8, EPI>), grid, dim3(kRowsThreads), 0, st, a);
      break;
    case 11:
      hipLaunchKernelGGL((gemm_rows16_kernel<6, EPI>), grid, dim3(kRowsThreads), 0, st, a);
      break;
    default: hipLaunchKernelGGL((gemm_kernel<4, 4, 4, 2, EPI>), grid, dim3(512), 0, st, a); break;
  }
  return hipGetLastError();
}

}  // namespace

// bf16: the smallest BM of {16, 32, 64, 256} that covers M (several M tiles
// past 256); the SwiGLU GEMM at BM 256 uses the 96-column tile. Split-K (1, 2, 4 or 8) only where allowed, to about one workgroup
// per CU, keeping an even number of at least 4 K steps per split.
GemmPlan plan_gemm(int dtype, int M, int N, int K, bool allow_split, bool swiglu, bool frag,
                   int max_splits) {
  GemmPlan p;
  constexpr int kCUs = 256;
  if (frag && !swiglu && dtype == LDR_BF16 && M > 64 && K % BK == 0) {
    // Activation rows in the fragment layout: 256 x BN tiles of 128, 96 or 64
    // columns and a K split of 1 .. 8 that keeps the workgroups within one
    // round over the CUs (no split where the tiles alone take more). Taken in
    // order: the plan whose workgroups fill the most of their last round; then
    // one whose K range is at most 2048 (longer ranges measured slower, each
    // workgroup re-reading more activation rows); then the fewest splits (the
    // fp32 partial tiles are written in a burst at the end and read back by
    // the next kernel); then the fewest bytes per workgroup.
    const int cands[3][2] = {{7, 128}, {6, 96}, {8, 64}};
    double best_u = -1.0, best_v = 0.0;
    bool best_short = false;
    for (const auto& c : cands) {
      const long tiles = (long)((N + c[1] - 1) / c[1]) * ((M + 255) / 256);
      for (int sp = 1; sp <= (allow_split ? max_splits : 1); sp *= 2) {
        if (K % (sp * BK) != 0 || K / sp < 2 * BK) break;
        const long wg = tiles * sp;
        if (sp > 1 && wg > kCUs) break;
        const double u = (double)wg / (double)(((wg + kCUs - 1) / kCUs) * kCUs);
        const bool shrt = K / sp <= 2048;
        const double vol = (256.0 + c[1]) * (K / sp) * 2.0;
        bool take;
        if (u > best_u + 1e-9) take = true;
        else if (u < best_u - 1e-9) take = false;
        else if (shrt != best_short) take = shrt;
        else if (sp != p.splits) take = sp < p.splits;
        else take = vol < best_v;
        if (take) {
          best_u = u; best_v = vol; best_short = shrt; p.cfg = c[0]; p.splits = sp;
          p.grid_x = (N + c[1] - 1) / c[1]; p.grid_y = (M + 255) / 256;
        }
      }
    }
    if (best_u > 0.0) { p.ntw = 0; return p; }
  }
  int bm, bn, kstep;
  if (dtype == LDR_F32) {
    p.cfg = -1; bm = 32; bn = 64; kstep = 16;
  } else {
    p.cfg = M <= 16 ? 0 : M <= 32 ? 1 : M <= 64 ? 2 : swiglu ? 4 : 3;
    if (p.cfg == 4) {
      // SwiGLU tiles (no split-K): the column width whose rounds over the CUs
      // times the bytes a tile streams (all its activation rows plus its
      // weight columns) is least, among 96 (cfg 4), 128 (cfg 3) and 64 (cfg 5)
      const int mt = (M + 255) / 256;
      double best = 0.0;
      const int cands[3][2] = {{4, 96}, {3, 128}, {5, 64}};
      for (const auto& c : cands) {
        const long tiles = (long)mt * ((N + c[1] - 1) / c[1]);
        const double cost = (double)((tiles + kCUs - 1) / kCUs) * (256.0 + c[1]) * K;
        if (best == 0.0 || cost < best) { best = cost; p.cfg = c[0]; }
      }
    }
    // the SwiGLU GEMM above 64 rows reads its rows in the fragment layout
    if (swiglu && M > 64 && K % BK == 0) p.cfg = p.cfg == 4 ? 6 : p.cfg == 3 ? 7 : p.cfg;
    if (p.cfg == 3 && allow_split && !swiglu) {
      const int t128 = ((N + 127) / 128) * ((M + 255) / 256);
      if (t128 * 8 <= kCUs && t128 * 16 > kCUs && K / 8 <= 512 && K % (4 * 2 * 2 * BK) == 0)
        p.cfg = 5;
    }
    bm = p.cfg >= 3 ? 256 : 16 << p.cfg;
    bn = p.cfg == 5 ? 64 : (p.cfg == 4 || p.cfg == 6) ? 96
         : (p.cfg == 3 || p.cfg == 0 || p.cfg == 7) ? 128 : 256;
    kstep = 2 * BK;
  }
  // split-K factor for `tiles` tiles: up to about one workgroup per CU, an
  // even number of at least 2 K steps per split
  auto split_for = [&](long tiles) {
    int s = 1;
    if (allow_split)
      while (s < max_splits && tiles * s * 2 <= kCUs && K % (2 * s * kstep) == 0 &&
             K / (2 * s) >= 2 * kstep)
        s *= 2;
    return s;
  };
  if (p.cfg == 0) {
    // 16-row tiles of 128 columns (4 waves) or 96 columns (cfg 9, 3 waves):
    // the width whose workgroups fill more of their last round over the CUs
    // (128 on a tie). At batch 1 the SwiGLU GEMM's 24576 columns make 192
    // tiles of 128 but 256 of 96 (47.6 and 47.7 us: these tiles stream their
    // weights at the chip's rate either way), and the QKV projection 48 x 4
    // against 64 x 4 (14.6 -> 13.2 us).
    auto fill = [&](int w) {
      const long tiles = (long)((N + w - 1) / w) * ((M + 15) / 16);
      const long wg = tiles * split_for(tiles);
      return (double)wg / (double)(((wg + kCUs - 1) / kCUs) * kCUs);
    };
    if (fill(96) > fill(128) + 1e-9) { p.cfg = 9; bn = 96; }
  }
  p.ntw = 0;
  p.grid_x = (N + bn - 1) / bn;
  p.grid_y = (M + bm - 1) / bm;
  p.splits = split_for((long)p.grid_x * p.grid_y);
  // 16-row tiles stream their weights through the loader waves' DMA
  if ((p.cfg == 0 || p.cfg == 9) && (K / p.splits) % BK == 0) p.cfg = p.cfg == 0 ? 10 : 11;
  return p;
}

hipError_t launch_gemm(int dtype, int epi, const GemmPlan& p, const GemmArgs& a,
                       hipStream_t st) {
  if (dtype == LDR_F32) {
    const dim3 grid(p.grid_x, p.grid_y, p.splits);
    if (epi == EPI_SWIGLU)
      hipLaunchKernelGGL((gemm_f32_kernel<EPI_SWIGLU>), grid, dim3(256), 0, st, a);
    else  // EPI_STORE and EPI_LOGITS share the fp32 store
      hipLaunchKernelGGL((gemm_f32_kernel<EPI_STORE>), grid, dim3(256), 0, st, a);
    return hipGetLastError();
  }
  const dim3 grid(p.grid_x, p.grid_y, p.splits);
  if (epi == EPI_SWIGLU) return launch_cfg<EPI_SWIGLU>(p.cfg, grid, a, st);
  if (epi == EPI_LOGITS) return launch_cfg<EPI_LOGITS>(p.cfg, grid, a, st);
  return launch_cfg<EPI_STORE>(p.cfg, grid, a, st);
}

bool gemm_tiled_supported(int M, int N, int K) {
  return M > 0 && N > 0 && K % (TK * 4) == 0;
}

hipError_t launch_gemm_tiled(const GemmArgs& a0, hipStream_t st) {
  if (!gemm_tiled_supported(a0.M, a0.N, a0.K) || a0.splits != 1) return hipErrorInvalidValue;
  GemmArgs a = a0;
  a.ldw = (a.N + TR - 1) / TR * TR;   // padded rows of a weight column block
  const dim3 grid((a.N + HB - 1) / HB, (a.M + TR - 1) / TR, 1);
  hipLaunchKernelGGL((gemm_tiled_kernel<kHeadLogits>), grid, dim3(512), 0, st, a,
                     HeadSampleArgs{});
  return hipGetLastError();
}

size_t head_sample_part_bytes(int rows, int vocab) {
  return (size_t)rows * ((vocab + HB - 1) / HB) * sizeof(HeadPart);
}

hipError_t launch_gemm_tiled_argmax(const GemmArgs& a0, const HeadSampleArgs& hs0, int32_t* tokens,
                                    float* lse, float* logq, hipStream_t st) {
  if (!gemm_tiled_supported(a0.M, a0.N, a0.K) || a0.splits != 1) return hipErrorInvalidValue;
  GemmArgs a = a0;
  a.ldw = (a.N + TR - 1) / TR * TR;
  HeadSampleArgs hs = hs0;
  hs.nparts = (a.N + HB - 1) / HB;
  const dim3 grid(hs.nparts, (a.M + TR - 1) / TR, 1);
  hipLaunchKernelGGL((gemm_tiled_kernel<kHeadArgmax>), grid, dim3(512), 0, st, a, hs);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(head_argmax_merge_kernel, dim3(a.M), dim3(64), 0, st,
                     static_cast<const HeadPart*>(hs.parts), hs.nparts, tokens, lse, logq);
  return hipGetLastError();
}

hipError_t launch_gemm_tiled_chunks(const GemmArgs& a0, const HeadSampleArgs& hs0,
                                    hipStream_t st) {
  if (!gemm_tiled_supported(a0.M, a0.N, a0.K) || a0.splits != 1 || !a0.out || !hs0.L ||
      !(hs0.T > 0.f) || hs0.ldL < (a0.N + 15) / 16)
    return hipErrorInvalidValue;
  GemmArgs a = a0;
  a.ldw = (a.N + TR - 1) / TR * TR;
  HeadSampleArgs hs = hs0;
  hs.store_logits = 1;
  const dim3 grid((a.N + HB - 1) / HB, (a.M + TR - 1) / TR, 1);
  if (hs.T == 1.f)
    hipLaunchKernelGGL((gemm_tiled_kernel<kHeadChunksUnitT>), grid, dim3(512), 0, st, a, hs);
  else
    hipLaunchKernelGGL((gemm_tiled_kernel<kHeadChunks>), grid, dim3(512), 0, st, a, hs);
  return hipGetLastError();
}

size_t tiled_elems(long rows, long cols) { return (size_t)((rows + TR - 1) / TR) * TR * cols; }

hipError_t launch_tile_matrix(const void* src, long ld, int rows, int cols, void* dst,
                              hipStream_t st) {
  const long chunks = (long)tiled_elems(rows, cols) / 8;
  const long want = (chunks + 255) / 256, blocks = want < 8192 ? want : 8192;
  const long R = (rows + TR - 1) / TR * TR;
  hipLaunchKernelGGL(tile_matrix_kernel, dim3((unsigned)blocks), dim3(256), 0, st,
                     static_cast<const uint16_t*>(src), ld, rows, R,
                     static_cast<uint16_t*>(dst), chunks);
  return hipGetLastError();
}

}  // namespace ldr
