// Weight-streaming GEMMs of the drafter: C[M][N] = A[M][K] . W[N][K]^T with
// fp32 accumulation, for the boundary fusion, the QKV / O / gate-up / down
// projections of every layer and the vocabulary head (Sec. 2.3, App. B.1).
//
// bf16: LDS-staged tiles feed v_mfma_f32_16x16x32_bf16. A workgroup owns a
// BM x BN output tile and a 1/splits share of K; the tiles of A and W for the
// next 64-wide K step are fetched into registers while the MFMAs consume the
// current one (two LDS buffers, one barrier per step). Rows of both operands
// are K-contiguous, so every lane's MFMA fragment is one 16-byte LDS read.
// fp32: a plain SIMT tile kernel with the same epilogues.
//
// Epilogues: EPI_STORE writes fp32 (split-K partials, or the logits when
// splits = 1); EPI_SWIGLU reads the gate and up rows of w_gate_up interleaved
// in 16-row blocks so that each lane holds matching gate/up sums, and writes
// silu(gate) * up in the activation dtype.
#include "ldr_internal.h"

namespace ldr {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int BK = 64;        // K step per LDS stage
constexpr int LDK = BK + 8;   // padded LDS row (elements): 144 B, conflict-free 16-lane reads

// Interleaved N index of the SwiGLU GEMM -> row of w_gate_up.
__device__ inline int swiglu_row(int c, int mlp) {
  const int blk = c >> 4, out = ((blk >> 1) << 4) | (c & 15);
  return (blk & 1) ? mlp + out : out;
}

__device__ inline float silu(float x) { return x / (1.f + expf(-x)); }

template <int BM, int BN, int WM, int WN, int EPI>
__global__ void __launch_bounds__(WM * WN * 64) gemm_bf16_kernel(GemmArgs a) {
  constexpr int NTHR = WM * WN * 64;
  constexpr int TM = BM / WM, TN = BN / WN, MT = TM / 16, NT = TN / 16;
  constexpr int ACH = BM * (BK / 8), WCH = BN * (BK / 8);  // 16-byte chunks per tile
  constexpr int AL = (ACH + NTHR - 1) / NTHR, WL = (WCH + NTHR - 1) / NTHR;
  static_assert(MT >= 1 && NT >= 1, "wave tile");
  static_assert(EPI != EPI_SWIGLU || (TN % 32) == 0, "swiglu pairs");
  __shared__ __attribute__((aligned(16))) uint16_t As[2][BM * LDK];
  __shared__ __attribute__((aligned(16))) uint16_t Ws[2][BN * LDK];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int n0 = blockIdx.x * BN, m0 = blockIdx.y * BM, z = blockIdx.z;
  const int kper = a.K / a.splits, kbeg = z * kper, nk = kper / BK;
  const uint16_t* A = static_cast<const uint16_t*>(a.A);
  const uint16_t* W = static_cast<const uint16_t*>(a.W);

  // Per-thread global source rows (fixed over K).
  const uint16_t* asrc[AL];
  const uint16_t* wsrc[WL];
  int adst[AL], wdst[WL];
#pragma unroll
  for (int i = 0; i < AL; ++i) {
    const int c = tid + i * NTHR, row = c >> 3, col = (c & 7) * 8;
    const int gm = m0 + row;
    asrc[i] = (c < ACH && gm < a.M) ? A + (long)gm * a.lda + kbeg + col : nullptr;
    adst[i] = c < ACH ? row * LDK + col : -1;
  }
#pragma unroll
  for (int i = 0; i < WL; ++i) {
    const int c = tid + i * NTHR, row = c >> 3, col = (c & 7) * 8;
    const int gn = n0 + row;
    int wrow = -1;
    if (c < WCH && gn < a.N) wrow = EPI == EPI_SWIGLU ? swiglu_row(gn, a.mlp) : gn;
    wsrc[i] = wrow >= 0 ? W + (long)wrow * a.ldw + kbeg + col : nullptr;
    wdst[i] = c < WCH ? row * LDK + col : -1;
  }

  uint4 ar[AL], wr[WL];
  auto fetch = [&](int kt) {
#pragma unroll
    for (int i = 0; i < AL; ++i)
      ar[i] = asrc[i] ? *reinterpret_cast<const uint4*>(asrc[i] + kt * BK) : make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int i = 0; i < WL; ++i)
      wr[i] = wsrc[i] ? *reinterpret_cast<const uint4*>(wsrc[i] + kt * BK) : make_uint4(0, 0, 0, 0);
  };
  auto stash = [&](int buf) {
#pragma unroll
    for (int i = 0; i < AL; ++i)
      if (adst[i] >= 0) *reinterpret_cast<uint4*>(&As[buf][adst[i]]) = ar[i];
#pragma unroll
    for (int i = 0; i < WL; ++i)
      if (wdst[i] >= 0) *reinterpret_cast<uint4*>(&Ws[buf][wdst[i]]) = wr[i];
  };

  f32x4 acc[MT][NT];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NT; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  fetch(0);
  stash(0);
  __syncthreads();
  int buf = 0;
  const int frow = lane & 15, fcol = (lane >> 4) * 8;
  for (int kt = 0; kt < nk; ++kt) {
    if (kt + 1 < nk) fetch(kt + 1);
#pragma unroll
    for (int kk = 0; kk < BK / 32; ++kk) {
      bf16x8 af[MT], bfr[NT];
#pragma unroll
      for (int i = 0; i < MT; ++i)
        af[i] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(
            &As[buf][(wm * TM + i * 16 + frow) * LDK + kk * 32 + fcol]));
#pragma unroll
      for (int j = 0; j < NT; ++j)
        bfr[j] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(
            &Ws[buf][(wn * TN + j * 16 + frow) * LDK + kk * 32 + fcol]));
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < NT; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) stash(buf ^ 1);
    __syncthreads();
    buf ^= 1;
  }

  // C layout of a 16x16 tile: lane holds rows (lane/16)*4 + v, column lane%16.
  const int crow = (lane >> 4) * 4, ccol = lane & 15;
  if constexpr (EPI == EPI_STORE) {
    float* out = static_cast<float*>(a.out) + (long)z * a.split_stride;
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < NT; ++j) {
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
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < NT; j += 2) {
        const int col = (n0 + wn * TN + j * 16) / 2 + ccol;
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

struct TileCfg { int BM, BN; };
constexpr TileCfg kCfg[3] = {{32, 64}, {64, 128}, {256, 128}};

template <int EPI>
hipError_t launch_bf16(const GemmPlan& p, const GemmArgs& a, hipStream_t st) {
  const dim3 grid(p.grid_x, p.grid_y, p.splits);
  switch (p.cfg) {
    case 0: hipLaunchKernelGGL((gemm_bf16_kernel<32, 64, 2, 2, EPI>), grid, dim3(256), 0, st, a); break;
    case 1: hipLaunchKernelGGL((gemm_bf16_kernel<64, 128, 1, 4, EPI>), grid, dim3(256), 0, st, a); break;
    default: hipLaunchKernelGGL((gemm_bf16_kernel<256, 128, 4, 2, EPI>), grid, dim3(512), 0, st, a); break;
  }
  return hipGetLastError();
}

}  // namespace

GemmPlan plan_gemm(int dtype, int M, int N, int K, bool allow_split) {
  GemmPlan p;
  int bm, bn;
  if (dtype == LDR_F32) {
    p.cfg = -1; bm = 32; bn = 64;
  } else {
    p.cfg = M <= 32 ? 0 : (M <= 64 ? 1 : 2);
    bm = kCfg[p.cfg].BM; bn = kCfg[p.cfg].BN;
  }
  p.grid_x = (N + bn - 1) / bn;
  p.grid_y = (M + bm - 1) / bm;
  const int kstep = dtype == LDR_F32 ? 16 : BK;
  int s = 1;
  if (allow_split) {
    const int tiles = p.grid_x * p.grid_y;
    while (tiles * s < 256 && s < 16 && K % (2 * s * kstep) == 0 && K / (2 * s) >= 256) s *= 2;
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
    else
      hipLaunchKernelGGL((gemm_f32_kernel<EPI_STORE>), grid, dim3(256), 0, st, a);
    return hipGetLastError();
  }
  return epi == EPI_SWIGLU ? launch_bf16<EPI_SWIGLU>(p, a, st) : launch_bf16<EPI_STORE>(p, a, st);
}

}  // namespace ldr
