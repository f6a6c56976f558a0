// Internal declarations of the drafting-step library: derived shapes, the
// per-sequence arena layout, bf16 helpers and the kernel launchers that the
// host API (api.cpp) calls. Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/ldr.h"

namespace ldr {

constexpr size_t kAlign = 256;
inline size_t align_up(size_t x, size_t a = kAlign) { return (x + a - 1) / a * a; }

// Byte offsets of the views inside one sequence's arena slot.
struct Layout {
  size_t kw, vw, m, eta, h;  // region offsets
  size_t ps;                 // fp32 sums of the pooled banks' open chunks
  size_t bytes;              // sum of the (aligned) regions
  size_t stride;             // per-sequence stride, bytes rounded up to kAlign
};

struct Shape {
  int hidden, hq, hkv, d, mlp, vocab, D, Lb, B, W, R, dtype;
  int rep;       // hq / hkv
  int qkv_out;   // (hq + 2 hkv) d
  float eps;
  double rope_base;
  size_t el;     // bytes per element of the configuration dtype
  bool keep_win, keep_sum, keep_bnd;  // views kept (ablation variants drop some)
  bool learned;  // the learned-query summary (Eq. 5) is kept
  int P, S0, S1; // mean-pooled summary: slots per bank and the two strides (P = 0: none)
  int Wr, Wx;    // window ring rows kept (W or 0) and rows per (layer, group): Wr + 2P
};

bool make_shape(const ldr_config* c, Shape* s);
Layout make_layout(const Shape& s);

// ---- bf16 helpers (round to nearest even, as torch does) ------------------
__host__ __device__ inline float bf16_to_f32(uint16_t h) {
  union { uint32_t u; float f; } v;
  v.u = (uint32_t)h << 16;
  return v.f;
}
// Lane swap inside a row of 16 lanes (DPP control CTRL: 0xB1 / 0x4E quad
// permutations xor 1 / xor 2, 0x141 half-row mirror, 0x140 row mirror).
template <int CTRL> __device__ inline float dpp(float v) {
#if defined(__HIP_DEVICE_COMPILE__)
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), CTRL,
                                                            0xF, 0xF, false));
#else
  return v;  // device code only
#endif
}

// Reductions over the 16 lanes of a row group with DPP lane swaps: quad
// permutations (xor 1, xor 2), then half-row and row mirrors, which pair each
// lane with one of the other half; every lane ends with the same value.
__device__ inline float sum16(float v) {
  v += dpp<0xB1>(v);   // quad_perm [1, 0, 3, 2]
  v += dpp<0x4E>(v);   // quad_perm [2, 3, 0, 1]
  v += dpp<0x141>(v);  // row_half_mirror
  v += dpp<0x140>(v);  // row_mirror
  return v;
}
__device__ inline float max16(float v) {
  v = fmaxf(v, dpp<0xB1>(v));
  v = fmaxf(v, dpp<0x4E>(v));
  v = fmaxf(v, dpp<0x141>(v));
  v = fmaxf(v, dpp<0x140>(v));
  return v;
}

// Chunk log-mass of the two-level draw at T > 0 (Eq. 8): one term
// exp(zt - m) of a chunk's sum, and the chunk's log-mass m + log s. The same
// operations (no contraction) wherever L_c is formed, so the log-mass pass over
// stored logits and the vocabulary head's epilogue give the same bits when
// they also sum the 16 terms in the same balanced pairwise order. A token
// outside the support (zt = -inf) adds exp2(-inf) = 0; a chunk without one
// has m = -inf and L_c = -inf; a NaN logit makes its chunk's L_c NaN, which the
// chunk draw leaves out like -inf.
#if defined(__HIP_DEVICE_COMPILE__)
__device__ inline float chunk_term(float zt, float m) {
#pragma clang fp contract(off)
  return __builtin_amdgcn_exp2f((zt - m) * 1.44269504088896341f);
}
__device__ inline float chunk_log_mass(float m, float s) {
#pragma clang fp contract(off)
  return m == -INFINITY ? -INFINITY : m + __builtin_amdgcn_logf(s) * 0.693147180559945309f;
}
#else
__device__ float chunk_term(float zt, float m);   // device code only
__device__ float chunk_log_mass(float m, float s);
#endif

// Round to nearest even (the device uses the gfx950 conversion instruction).
__host__ __device__ inline uint16_t f32_to_bf16(float f) {
#if defined(__HIP_DEVICE_COMPILE__)
  return __builtin_bit_cast(uint16_t, (__bf16)f);
#else
  union { uint32_t u; float f; } v;
  v.f = f;
  if ((v.u & 0x7f800000u) == 0x7f800000u && (v.u & 0x007fffffu))  // NaN stays NaN
    return (uint16_t)((v.u >> 16) | 0x40);
  uint32_t r = v.u + 0x7fffu + ((v.u >> 16) & 1u);
  return (uint16_t)(r >> 16);
#endif
}

// Workgroup barrier that orders LDS accesses only: each wave waits for its own
// LDS operations, not for its global loads still in flight. __syncthreads()
// also drains every outstanding global load, which would stall software
// pipelines that keep prefetches in flight across the barrier. Register data
// from those loads is still waited for where it is consumed.
__device__ inline void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

template <typename T> struct Elem;
template <> struct Elem<float> {
  __device__ static float load(const float* p) { return *p; }
  __device__ static void store(float* p, float v) { *p = v; }
};
template <> struct Elem<uint16_t> {
  __device__ static float load(const uint16_t* p) { return bf16_to_f32(*p); }
  __device__ static void store(uint16_t* p, float v) { *p = f32_to_bf16(v); }
};

// Top-k support of a row of logits: token v is inside iff order_key(z_v) > tau,
// or order_key(z_v) == tau and v <= v_cut (ties at the boundary, lower index
// first).
struct TopK { uint32_t tau; int v_cut; };

// Order-preserving map of fp32 to uint32 (larger float, larger key); -0
// counts as +0, as the two compare equal.
__device__ inline uint32_t order_key(float z) {
  uint32_t b = __float_as_uint(z);
  if (b == 0x80000000u) b = 0u;
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}
__device__ inline bool in_support(const TopK& t, float z, int v) {
  const uint32_t u = order_key(z);
  return u > t.tau || (u == t.tau && v <= t.v_cut);
}

// ---- kernel launchers -------------------------------------------------------
// Views (views.hip)
hipError_t launch_views_reset(const Shape& s, const Layout& L, int batch, void* arena,
                              int64_t* pos, hipStream_t st);
// done: a device counter (0 between launches) when this launch commits
// (advances pos, or flags a bad count in status) from its last workgroup;
// null when a later launch reads pos and commits instead.
hipError_t launch_views_update(const Shape& s, const Layout& L, int batch, void* arena,
                               int64_t* pos, const void* G, const int32_t* n_new,
                               int max_new, const void* K_new, const void* V_new,
                               const void* h_new, hipStream_t st, int32_t* status,
                               int32_t* done);
// Mean-pooled summary banks (views.hip); runs after the update, before the
// commit (done as above).
hipError_t launch_views_pool(const Shape& s, const Layout& L, int batch, void* arena,
                             int64_t* pos, const int32_t* n_new, int max_new,
                             const void* K_new, const void* V_new, hipStream_t st,
                             int32_t* status, int32_t* done);
// Without new rows (no update launch): the commit alone.
hipError_t launch_views_commit(int batch, int64_t* pos, const int32_t* n_new, int max_new,
                               int32_t* status, hipStream_t st);

// GEMM (gemm.hip): C = A[M][K] . W[N][K]^T, fp32 accumulation.
enum GemmEpi {
  EPI_STORE = 0,   // out fp32 [split][M][N] (split-K partials; split 0 only if S = 1)
  EPI_SWIGLU = 1,  // W rows are [gate; up] (N = 2 mlp): act[M][mlp] = silu(g) * u
  EPI_LOGITS = 2,  // the vocabulary head: fp32 logits [M][V], never split
};
struct GemmArgs {
  const void* A; long lda;     // [M][K] activations (dtype), row stride in elements
  const void* W; long ldw;     // [N][K] weights (dtype)
  void* out;                   // EPI_STORE: float*; EPI_SWIGLU: dtype*
  long ldo;                    // output row stride (elements)
  long split_stride;           // EPI_STORE: elements between split partials
  int M, N, K, splits;
  int mlp;                     // EPI_SWIGLU: N / 2
  int out_frag = 0;            // EPI_SWIGLU: output [M][mlp] in the fragment layout
};
struct GemmPlan { int cfg, ntw, splits; int grid_x, grid_y; };  // cfg: tile configuration
// The plan's kernel reads its activation rows in the fragment layout (NRM_FRAG).
inline bool gemm_plan_frag(const GemmPlan& p) { return p.cfg >= 6 && p.cfg <= 8; }
// Tile configuration and split-K factor; splits = 1 unless allow_split, at
// most max_splits (a power of two). frag: the caller can give the activation
// rows in the fragment layout.
GemmPlan plan_gemm(int dtype, int M, int N, int K, bool allow_split, bool swiglu = false,
                   bool frag = false, int max_splits = 8);
hipError_t launch_gemm(int dtype, int epi, const GemmPlan& p, const GemmArgs& a, hipStream_t st);
// bf16 GEMM for the vocabulary head: A in 256-row tiles of 32-column blocks
// (the final norm's tiled output), W [N][K] in the column-block layout of
// ldr_tile_matrix; fp32 out [M][ldo]. Needs K % 128 == 0 and splits == 1.
bool gemm_tiled_supported(int M, int N, int K);
hipError_t launch_gemm_tiled(const GemmArgs& a, hipStream_t st);
// The vocabulary head with greedy sampling (T = 0) fused into its epilogue:
// per row and column tile the first argmax goes to `parts`, then one merge per
// row writes the token, lse (its logit) and log q = 0. The logits are written
// only if store_logits.
struct HeadSampleArgs {
  void* parts;        // head_sample_part_bytes(M, V) bytes
  int nparts;         // partials per row (set by the launcher)
  int store_logits;
  float* L;           // T > 0: chunk log-masses [M][ldL] (the sampler's layout)
  int ldL;
  float T;
};
size_t head_sample_part_bytes(int rows, int vocab);
hipError_t launch_gemm_tiled_argmax(const GemmArgs& a, const HeadSampleArgs& hs, int32_t* tokens,
                                    float* lse, float* logq, hipStream_t st);
// The vocabulary head at T > 0 with the first level of the two-level draw in
// its epilogue: it writes the logits and every 16-token chunk's log-mass
// L_c = log sum exp(z / T) to hs.L, bit for bit what the sampler's log-mass
// pass forms from the written logits; the chunk draw then follows as in the
// sampler.
hipError_t launch_gemm_tiled_chunks(const GemmArgs& a, const HeadSampleArgs& hs, hipStream_t st);
// Elements of a [rows][cols] matrix in the tiled layout (rows padded to 256).
size_t tiled_elems(long rows, long cols);
hipError_t launch_tile_matrix(const void* src, long ld, int rows, int cols, void* dst,
                              hipStream_t st);

// Draft step pieces (draft.hip)
struct DraftPtrs {
  const uint8_t* arena; const int64_t* pos; const void* G;
  float* part;     // split-K partials
  float* x;        // residual stream fp32 [M][hidden]
  void* nrm;       // normalised activations (dtype) [M][hidden]
  void* qkv;       // block q, k, v after RMSNorm and RoPE (dtype) [M][qkv_out]
  void* o;         // attention output (dtype) [M][hq d]
  void* act;       // SwiGLU output (dtype) [M][mlp]
  float* rope;     // cos/sin [batch][B][d/2] x 2
  int32_t* status; // sticky flags of the views handle
};

// Bits of the sticky device status word.
constexpr int kFlagRange = 1;   // an update saw a row count outside [0, max_new]
constexpr int kFlagAnchor = 2;  // a draft step saw an anchor outside [0, V)
// Word of the views' 256-byte status block (its own 64-byte line) that counts
// the workgroups of an update launch done (0 between launches).
constexpr int kCommitCounter = 16;
// Attention over [block; window; summary] of one layer (Eq. 6).
struct AttnArgs {
  const void* qkv;   // block q, k, v rows (dtype) [M][qkv_out], normalised and rotated
                     // (vector kernel)
  // bf16 kernel: the QKV projection's fp32 split-K partials [splits][rows][qkv_out]
  // and what finishing them takes (q / k RMSNorm gains, the RoPE table
  // cos / sin [rows][d/2] x 2, eps)
  const float* part; long split_stride; int splits, rows;
  const void* q_norm; const void* k_norm; const float* rope; float eps;
  const uint8_t* arena; size_t stride; size_t kw, vw, m_off;
  const int64_t* pos; const void* G;
  void* o;
  int layer, hq, hkv, d, B, W, R, rep, qkv_out;
  int Wx;            // rows per (layer, group) region: the W window rows (0 if
                     // dropped), then 2P pooled slot means
  int P, S0, S1;     // mean-pooled summary (P = 0: none)
  int use_summary;   // the learned summary is kept
  float inv_sqrt_d;
  int o_frag;        // o in the fragment layout of [M][hq d] (bf16 kernel), else row-major
};
// bf16 MFMA kernel (attn.hip): one workgroup per (kv group, sequence).
hipError_t launch_attention_mfma(const AttnArgs& a, int hkv, int batch, hipStream_t st);
bool attention_mfma_supported(int d, int rep, int B, int R, int Wx);

// frag_out: write layer 0's normalised rows there in the fragment layout
// instead of to p.nrm.
hipError_t launch_slot_init(const Shape& s, int batch, const DraftPtrs& p, int fc_splits,
                            const ldr_weights* w, const int32_t* anchor, hipStream_t st,
                            void* frag_out = nullptr);
bool norm_hidden_supported(int hidden);
// Layouts of the normalised rows a residual norm writes.
enum NrmLayout {
  NRM_ROWS = 0,   // row-major [M][hidden] (p.nrm)
  NRM_TILED = 1,  // 256-row x 32-column blocks (the tiled vocabulary head's activation rows)
  NRM_FRAG = 2,   // 16-row x 32-column MFMA fragments, lane order (gemm_frag_kernel)
};
// tiled_out: write the normalised rows there in `layout` instead of to p.nrm.
hipError_t launch_resid_norm(const Shape& s, int M, const DraftPtrs& p, int splits,
                             const void* gain, hipStream_t st, void* tiled_out = nullptr,
                             int layout = NRM_TILED);
// fp32 models only (the bf16 attention kernel finishes q, k, v itself).
hipError_t launch_qkv_finish(const Shape& s, int M, const DraftPtrs& p, int splits,
                             const ldr_layer_weights* lw, hipStream_t st);
// o_frag: the output in the fragment layout (bf16 only).
// bf16: the kernel also finishes q, k and v from the QKV partials (qkv_splits
// of them, 1, 2 or 4; lw's q / k gains); the vector kernel reads p.qkv.
hipError_t launch_attention(const Shape& s, const Layout& L, int batch, const DraftPtrs& p,
                            int layer, const ldr_layer_weights* lw, int qkv_splits,
                            hipStream_t st, bool o_frag = false);

// Sampler (sample.hip)
// T = 0: greedy_splits chunks of greedy_chunk tokens per row. T > 0: nch
// chunks of 16 tokens per row, their log-masses in rows of ldL floats.
struct SamplePlan { int greedy_chunk, greedy_splits, nch, ldL; };
SamplePlan sample_plan(int rows, int vocab);
// Tokens per workgroup of the chunk log-mass pass over ntok tokens of `rows` rows.
int chunk_lse_slice(int rows, int ntok);
// The full-vocabulary sampler at T > 0 in pieces (top_k = 0): the chunk
// log-masses of tokens [v0, v1) of every row (v0 a multiple of 16), then,
// once all are written, the chunk keys and the in-chunk draw;
// ws as for launch_sample.
hipError_t launch_chunk_lse(const float* logits, int rows, int vocab, float temperature, void* ws,
                            int v0, int v1, hipStream_t st);
hipError_t launch_sample_finish(const float* logits, int rows, int vocab, float temperature,
                                uint64_t seed, uint64_t step, void* ws, int32_t* tokens,
                                float* lse, float* logq, hipStream_t st);
// Bytes of the sampler's workspace before its top-k supports: the chunk
// log-masses and the partials.
size_t sample_part_bytes(int rows, int vocab);
hipError_t launch_sample(const float* logits, int rows, int vocab, float temperature,
                         int top_k, uint64_t seed, uint64_t step, int32_t* tokens, float* lse,
                         float* logq, void* ws, size_t sel_off, hipStream_t st, int row_mul = 1,
                         int row_add = 0);
// Markov-corrected sampling of [batch][B][V] logits (corrected in place), one
// position after the other; ws / sel_off as for launch_sample with batch rows.
hipError_t launch_sample_markov(float* logits, int batch, int B, int vocab, const int32_t* anchor,
                                const void* E, const void* W, int rank, int dtype,
                                float temperature, int top_k, uint64_t seed, uint64_t step,
                                int32_t* tokens, float* lse, float* logq, void* ws,
                                size_t sel_off, hipStream_t st);
// Verification (verify.hip): Eq. 1-2 over [batch][B + 1][V] target logits.
size_t verify_workspace_bytes(int batch, int B, int V);
hipError_t launch_verify(const float* P, const float* z, const int32_t* y, const float* qlse,
                         int batch, int B, int V, float T, int top_k, uint64_t seed, uint64_t step,
                         int32_t* accepted, int32_t* token, int32_t* n_new, void* ws,
                         hipStream_t st);
// Top-k support (tau, v_cut) of each of `rows` rows of [rows][vocab] logits,
// 0 < k < vocab (sample.hip).
hipError_t launch_topk_select(const float* logits, int rows, int vocab, int k, TopK* sel,
                              hipStream_t st);
// Device address of the static scratch of ldr_sample_noalloc on the current
// GPU (sample.hip); looked up once per device.
hipError_t noalloc_scratch(void** out);
hipError_t launch_gumbel_fill(uint64_t seed, uint64_t step, int stream, int rows, int vocab,
                              float* out, hipStream_t st);

}  // namespace ldr
