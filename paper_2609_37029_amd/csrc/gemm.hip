// Weight-streaming GEMMs of the drafter: C[M][N] = A[M][K] . W[N][K]^T with
// fp32 accumulation, for the boundary fusion, the QKV / O / gate-up / down
// projections of every layer and the vocabulary head (Sec. 2.3, App. B.1).
//
// With M = batch x B rows (256 at batch 16) these GEMMs stream each weight
// once from HBM and reuse it across all M rows:
//  * a workgroup owns a BM x BN output tile (BM = all M rows up to 256) and a
//    1/splits share of K, with WM x WN waves of MTW x NTW 16x16 MFMA tiles;
//  * both operands reach LDS through coalesced 16-byte loads (8 lanes per
//    128-byte row segment), double-buffered, rows padded to 144 B so the
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
// and writes silu(gate) * up in the activation dtype.
#include "ldr_internal.h"

namespace ldr {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
// 16 bytes as a native vector (HIP's uint4 is a struct whose copies become
// memcpys that keep arrays of them in scratch).
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int BK = 64;        // K step: one LDS stage, two MFMA k-steps
constexpr int LDK = BK + 8;   // padded LDS row (elements): 144 B
constexpr int WPF = 4;        // weight steps in flight

// Interleaved N index of the SwiGLU GEMM -> row of w_gate_up.
__device__ inline int swiglu_row(int c, int mlp) {
  const int blk = c >> 4, out = ((blk >> 1) << 4) | (c & 15);
  return (blk & 1) ? mlp + out : out;
}

__device__ inline float silu(float x) { return x / (1.f + expf(-x)); }

template <int MTW, int NTW, int WM, int WN, int EPI>
__global__ void __launch_bounds__(WM * WN * 64, 1) gemm_kernel(GemmArgs a) {
  constexpr int NTHR = WM * WN * 64, TM = MTW * 16, TN = NTW * 16;
  constexpr int BM = WM * TM, BN = WN * TN;
  constexpr int ACH = BM * (BK / 8), WCH = BN * (BK / 8);   // 16-byte chunks per stage
  constexpr int AL = (ACH + NTHR - 1) / NTHR, WL = (WCH + NTHR - 1) / NTHR;
  static_assert(EPI != EPI_SWIGLU || NTW % 2 == 0, "swiglu pairs");
  __shared__ __attribute__((aligned(16))) uint16_t As[2][BM * LDK];
  __shared__ __attribute__((aligned(16))) uint16_t Ws[2][BN * LDK];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int n0 = blockIdx.x * BN, m0 = blockIdx.y * BM, z = blockIdx.z;
  const int kper = a.K / a.splits, kbeg = z * kper, nk = kper / BK;
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
    adst[i] = row * LDK + col;
  }
#pragma unroll
  for (int i = 0; i < WL; ++i) {
    const int c = (tid + i * NTHR) % WCH, row = c >> 3, col = (c & 7) * 8;
    const int gn = min(n0 + row, a.N - 1);
    const int wrow = EPI == EPI_SWIGLU ? swiglu_row(gn, a.mlp) : gn;
    wsrc[i] = W + (long)wrow * a.ldw + kbeg + col;
    wdst[i] = row * LDK + col;
  }

  // wq[p]: weights of step kt + 1 + p; a0 / a1: activation stages kt + 1 and
  // kt + 2 (roles swap every step). Constant indices only: registers.
  u32x4 wq[WPF][WL];
  u32x4 a0[AL], a1[AL];
  f32x4 acc[MTW][NTW];
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
              &Ws[buf][(wn * TN + j * 16 + (lane & 15)) * LDK + kk * 32 + (lane >> 4) * 8])); \
      _Pragma("unroll") for (int i = 0; i < MTW; ++i) {                               \
        const bf16x8 av = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>( \
            &As[buf][(wm * TM + i * 16 + (lane & 15)) * LDK + kk * 32 + (lane >> 4) * 8])); \
        _Pragma("unroll") for (int j = 0; j < NTW; ++j) acc[i][j] =                   \
            __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bfr[j], acc[i][j], 0, 0, 0);  \
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

  // C layout of a 16x16 tile: lane holds rows (lane/16)*4 + v, column lane%16.
  const int crow = (lane >> 4) * 4, ccol = lane & 15;
  if constexpr (EPI == EPI_STORE || EPI == EPI_LOGITS) {
    float* out = static_cast<float*>(a.out) + (long)z * a.split_stride;
#pragma unroll
    for (int i = 0; i < MTW; ++i)
#pragma unroll
      for (int j = 0; j < NTW; ++j) {
        const int col = n0 + wn * TN + j * 16 + ccol;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int row = m0 + wm * TM + i * 16 + crow + v;
          if (row < a.M && col < a.N) out[(long)row * a.ldo + col] = acc[i][j][v];
        }
      }
  } else {
    uint16_t* out = static_cast<uint16_t*>(a.out);
#pragma unroll
    for (int j = 0; j < NTW; j += 2) {   // n-tiles j (gate) and j + 1 (up) of 16 output columns
      const int col = (n0 + wn * TN + j * 16) / 2 + ccol;
#pragma unroll
      for (int i = 0; i < MTW; ++i)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int row = m0 + wm * TM + i * 16 + crow + v;
          if (row < a.M && col < a.mlp)
            out[(long)row * a.ldo + col] = f32_to_bf16(silu(acc[i][j][v]) * acc[i][j + 1][v]);
        }
    }
  }
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

// Tile configurations (cfg): 0: BM 16 (M <= 16) with 4 waves along N (BN 128);
// 1: BM 32, 2: BM 64, with 8 waves along N (BN 256); 3: BM 256 with 4 x 2 waves
// of 64 x 64 (BN 128);
// 4: BM 256 with 8 x 1 waves of 32 x 96 (BN 96), for the SwiGLU GEMM, whose
// 2 x 12288 columns at the Qwen3-8B shape make exactly 256 tiles (one per CU).
template <int EPI>
hipError_t launch_cfg(int cfg, dim3 grid, const GemmArgs& a, hipStream_t st) {
  switch (cfg) {
    case 0: hipLaunchKernelGGL((gemm_kernel<1, 2, 1, 4, EPI>), grid, dim3(256), 0, st, a); break;
    case 1: hipLaunchKernelGGL((gemm_kernel<2, 2, 1, 8, EPI>), grid, dim3(512), 0, st, a); break;
    case 2: hipLaunchKernelGGL((gemm_kernel<4, 2, 1, 8, EPI>), grid, dim3(512), 0, st, a); break;
    case 4: hipLaunchKernelGGL((gemm_kernel<2, 6, 8, 1, EPI>), grid, dim3(512), 0, st, a); break;
    default: hipLaunchKernelGGL((gemm_kernel<4, 4, 4, 2, EPI>), grid, dim3(512), 0, st, a); break;
  }
  return hipGetLastError();
}

}  // namespace

// bf16: the smallest BM of {16, 32, 64, 256} that covers M (several M tiles
// past 256); the SwiGLU GEMM at BM 256 uses the 96-column tile. Split-K (1, 2, 4 or 8) only where allowed, to about one workgroup
// per CU, keeping an even number of at least 4 K steps per split.
GemmPlan plan_gemm(int dtype, int M, int N, int K, bool allow_split, bool swiglu) {
  GemmPlan p;
  constexpr int kCUs = 256;
  int bm, bn, kstep;
  if (dtype == LDR_F32) {
    p.cfg = -1; bm = 32; bn = 64; kstep = 16;
  } else {
    p.cfg = M <= 16 ? 0 : M <= 32 ? 1 : M <= 64 ? 2 : swiglu ? 4 : 3;
    bm = p.cfg >= 3 ? 256 : 16 << p.cfg;
    bn = p.cfg == 4 ? 96 : (p.cfg == 3 || p.cfg == 0) ? 128 : 256;
    kstep = 2 * BK;
  }
  p.ntw = 0;
  p.grid_x = (N + bn - 1) / bn;
  p.grid_y = (M + bm - 1) / bm;
  int s = 1;
  if (allow_split) {
    const int tiles = p.grid_x * p.grid_y;
    while (s < 8 && tiles * s * 2 <= kCUs && K % (2 * s * kstep) == 0 && K / (2 * s) >= 2 * kstep)
      s *= 2;
  }
  p.splits = s;
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

}  // namespace ldr
