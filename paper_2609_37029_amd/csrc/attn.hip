// Block-view attention on MFMA for bf16 views (Eq. 6; App. A.1; Sec. 2.4).
//
// One workgroup per (kv group g, sequence b, HPW query heads of the group),
// NSEG waves per head, each taking one segment of the key sources under its
// own online softmax: segment 0 the block's own k / v (B rows, normalised and
// rotated by the QKV finishing kernel) and the first window chunks, the last
// segment the last window chunks of layer j and the head's R summary entries
// (keys G[j,h], values M[j,h] rounded to bf16). Window chunks of 32 keys are
// staged through LDS once for all heads of the workgroup (K rows and the
// transposed V rows as stored in the views), fetched into registers ahead of
// use. The segments merge their (max, sum, O) in LDS, which is the split form
// of the one softmax over all sources. With 8 or more chunks and heads in
// pairs (the Qwen3 shapes) a workgroup takes 2 heads in 4 segments, so the
// batch-16 launch has 256 workgroups and every wave walks 2-3 items.
// S = Q K^T and O += P V run on v_mfma_f32_16x16x32_bf16 (16 query rows per
// wave = the B <= 16 slots); P goes through a per-wave LDS tile to change
// from the C layout to the A layout.
#include "ldr_internal.h"

namespace ldr {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int KC = 32;  // keys per chunk
constexpr int QR = 16;  // query rows per wave (block slots, zero-padded)

__device__ inline float sum64(float v) {
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
  return v;
}
__device__ inline bf16x8 frag(const uint16_t* p) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(p));
}
__device__ inline void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

// HPW query heads of one kv group per workgroup (a group with more heads
// spreads over rep / HPW workgroups, each reading the group's window), NSEG
// waves per head: the key sources are cut into NSEG segments, segment 0
// taking the block's own k / v and the first window chunks, segment NSEG - 1
// the last window chunks and the R summary entries; every wave keeps the
// online-softmax state of its segment, and the segments merge their
// (max, sum, O) in LDS at the end. Each segment stages its chunks through one
// LDS tile pair (K rows, V^T rows), two barriers per step.
template <int D, int HPW, int NSEG, int WD>
__global__ void __launch_bounds__(64 * HPW * NSEG) attention_mfma_kernel(AttnArgs a) {
  constexpr int NT = 64 * HPW * NSEG, ST = 64 * HPW;  // threads, threads per segment
  constexpr int LDQ = D + 8;   // bf16 row of the Q / K tiles (conflict-free 16-row reads)
  constexpr int LDV = KC + 8;  // bf16 row of the V^T / P tiles
  constexpr int NDT = D / 16, KS = D / 32;
  constexpr int CH = KC * D / 8;              // 16-byte pieces of one chunk matrix
  constexpr int PL = (CH + ST - 1) / ST;      // pieces per thread of its segment
  constexpr int RMAX = 16;
  constexpr int KTILE = KC * LDQ, VTILE = D * LDV, SEGT = KTILE + VTILE;
  // The tile area holds the segments' chunk tiles during the loop, then the
  // summary keys G and values M^T of the heads, then the merge data.
  constexpr int SUMT = HPW * (RMAX * LDQ + VTILE);
  constexpr int MERGE = (NSEG - 1) * HPW * (QR * D + 2 * QR) * 2;   // in bf16 units
  constexpr int AREA = NSEG * SEGT > SUMT ? (NSEG * SEGT > MERGE ? NSEG * SEGT : MERGE)
                                          : (SUMT > MERGE ? SUMT : MERGE);
  __shared__ __attribute__((aligned(16))) uint16_t Qs[HPW][QR * LDQ];
  __shared__ __attribute__((aligned(16))) uint16_t Tile[AREA];
  __shared__ __attribute__((aligned(16))) uint16_t Pt[HPW * NSEG][QR * LDV];
  uint16_t* const Gs = Tile;                          // [HPW][RMAX * LDQ]
  uint16_t* const Mt = Tile + HPW * RMAX * LDQ;       // [HPW][D * LDV]
  float* const Xo = reinterpret_cast<float*>(Tile);   // [NSEG - 1][HPW][QR][D]
  float* const Xml = Xo + (NSEG - 1) * HPW * QR * D;  // [NSEG - 1][HPW][QR][2]

  // blockIdx.x = head set * hkv + group: the workgroups that read one group's
  // window are hkv apart in the dispatch order, so with 8 kv groups they land
  // on the same XCD and share its L2
  const int g = blockIdx.x % a.hkv, b = blockIdx.y;
  const int h0 = g * a.rep + (blockIdx.x / a.hkv) * HPW;  // first head of the workgroup
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int seg = w / HPW, hh = w % HPW, h = h0 + hh;
  const int ht = threadIdx.x - seg * ST;  // thread index inside the segment
  uint16_t* const Ks = Tile + seg * SEGT;
  uint16_t* const Vt = Ks + KTILE;
  const int B = a.B;
  const uint8_t* seq = a.arena + (size_t)b * a.stride;
  const size_t gw = (size_t)(a.layer * a.hkv + g) * a.Wx * D;   // window rows, then pooled slots
  const uint16_t* Kw = reinterpret_cast<const uint16_t*>(seq + a.kw) + gw;
  const uint16_t* Vw = reinterpret_cast<const uint16_t*>(seq + a.vw) + gw;
  // window chunks of the segment, assigned over the full region so that the
  // first fetches do not wait for the position t (unfilled slots read as
  // zeros and are masked); the launcher keeps every segment nonempty
  const int nwf = a.Wx / KC;
  const int cbeg = seg * nwf / NSEG, cend = (seg + 1) * nwf / NSEG;

  // ---- block rows: q of the workgroup's heads, k and v of the group (already
  // normalised and rotated), zero past the B slots of the 16-row tile; k and v
  // go to segment 0's tiles.
  constexpr int QP = HPW * QR * D / 8, KP = QR * D / 8;  // 16-byte pieces
  constexpr int NP = QP + 2 * KP, PP = (NP + NT - 1) / NT;
  const uint16_t* qkv = static_cast<const uint16_t*>(a.qkv) + (size_t)b * B * a.qkv_out;
  u32x4 pre[PP];
#pragma unroll
  for (int i = 0; i < PP; ++i) {
    const int idx = threadIdx.x + i * NT;
    const int j = idx < QP ? idx % (QR * D / 8) : (idx - QP) % KP;
    const int row = j / (D / 8), c8 = (j % (D / 8)) * 8;
    const int col = idx < QP ? (h0 + idx / (QR * D / 8)) * D + c8
                  : idx < QP + KP ? (a.hq + g) * D + c8 : (a.hq + a.hkv + g) * D + c8;
    pre[i] = (idx < NP && row < B)
                 ? *reinterpret_cast<const u32x4*>(qkv + (size_t)row * a.qkv_out + col)
                 : u32x4{0u, 0u, 0u, 0u};
  }
  // Window chunks in flight: slot p of the ring holds the p-th next chunk of
  // the segment (depth WD, rotated by shifting), all issued before the first wait.
  u32x4 wk[WD][PL], wv[WD][PL];
#pragma unroll
  for (int p = 0; p < WD; ++p)
#pragma unroll
    for (int i = 0; i < PL; ++i) wk[p][i] = wv[p][i] = u32x4{0u, 0u, 0u, 0u};
  const bool win = a.Wx > 0;  // no window and no pooled summary: no rows to stage
#define LDR_FETCH(p, c)                                                                  \
  if (win) {                                                                             \
    _Pragma("unroll") for (int i = 0; i < PL; ++i) {                                     \
      const int idx_ = (ht + i * ST) % CH;                                               \
      const int slot_ = (c) * KC + idx_ / (D / 8), col_ = (idx_ % (D / 8)) * 8;          \
      wk[p][i] = *reinterpret_cast<const u32x4*>(Kw + (size_t)slot_ * D + col_);       \
      wv[p][i] = *reinterpret_cast<const u32x4*>(Vw + (size_t)(idx_ >> 2) * a.Wx +      \
                                                 (c) * KC + (idx_ & 3) * 8);             \
    }                                                                                    \
  }
  int nf = cbeg;  // next chunk to fetch (clamped to the segment's last chunk)
#pragma unroll
  for (int p = 0; p < WD; ++p) { LDR_FETCH(p, max(0, min(nf, cend - 1))) ++nf; }

  // Summary keys and values of the workgroup's heads: loaded now, kept in
  // registers through the loop and parked in LDS after it. Rows past R are 0.
  constexpr int SG = HPW * RMAX * D / 8;      // 16-byte pieces of G (bf16)
  constexpr int SM = HPW * RMAX * D / 4;      // 16-byte pieces of M (fp32)
  constexpr int GL = (SG + NT - 1) / NT, ML = (SM + NT - 1) / NT;
  uint4 greg[GL], mreg[ML];
  {
    const size_t hrow = (size_t)(a.layer * a.hq + h0) * a.R;  // first row of the workgroup
    const uint16_t* Gg = static_cast<const uint16_t*>(a.G) + hrow * D;
    const float* Mg = reinterpret_cast<const float*>(seq + a.m_off) + hrow * D;
#pragma unroll
    for (int i = 0; i < GL; ++i) {
      const int idx = threadIdx.x + i * NT;
      const int hq_ = idx / (RMAX * D / 8), r = (idx / (D / 8)) % RMAX, col = (idx % (D / 8)) * 8;
      greg[i] = (a.use_summary && idx < SG && r < a.R)
                    ? *reinterpret_cast<const uint4*>(Gg + ((size_t)hq_ * a.R + r) * D + col)
                    : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < ML; ++i) {
      const int idx = threadIdx.x + i * NT;
      const int hq_ = idx / (RMAX * D / 4), r = idx % RMAX, col = ((idx / RMAX) % (D / 4)) * 4;
      mreg[i] = (a.use_summary && idx < SM && r < a.R)
                    ? *reinterpret_cast<const uint4*>(Mg + ((size_t)hq_ * a.R + r) * D + col)
                    : make_uint4(0, 0, 0, 0);
    }
  }

  const long t = a.pos[b];
  const int nv = t < a.W ? (int)t : a.W;   // valid window rows (W = 0 without the window)
  // Mean-pooled summary: its banks' slots follow the window rows; slot k of a
  // bank is valid once k chunks have begun. Every chunk of the region is then
  // walked (the ones without a valid row are skipped), as at steady state.
  int np0 = 0, np1 = 0;
  if (a.P) {
    np0 = (int)min((t + a.S0 - 1) / a.S0, (long)a.P);
    np1 = (int)min((t + a.S1 - 1) / a.S1, (long)a.P);
  }
  auto chunk_valid = [&](int chunk) -> int {   // valid rows of a 32-row chunk
    const int r0 = chunk * KC;
    const int v = r0 < a.W ? nv - r0 : r0 < a.W + a.P ? np0 - (r0 - a.W) : np1 - (r0 - a.W - a.P);
    return v < 0 ? 0 : v > KC ? KC : v;
  };
  const int nwin = a.P ? nwf : (nv + KC - 1) / KC;
  // items of a segment: its window chunks below nwin, and the block for segment 0
  auto seg_items = [&](int sg) -> int {
    const int c0 = sg * nwf / NSEG, c1 = (sg + 1) * nwf / NSEG;
    return (sg == 0 ? 1 : 0) + max(0, min(nwin, c1) - c0);
  };
  const int items = seg_items(seg);
  int steps = 0;   // the same on every thread: every wave meets every barrier
#pragma unroll
  for (int sg = 0; sg < NSEG; ++sg) steps = max(steps, seg_items(sg));
#pragma unroll
  for (int i = 0; i < PP; ++i) {
    const int idx = threadIdx.x + i * NT;
    if (idx >= NP) break;
    const int j = idx < QP ? idx % (QR * D / 8) : (idx - QP) % KP;
    const int row = j / (D / 8), c8 = (j % (D / 8)) * 8;
    if (idx < QP) {
      *reinterpret_cast<u32x4*>(&Qs[idx / (QR * D / 8)][row * LDQ + c8]) = pre[i];
    } else if (idx < QP + KP) {
      *reinterpret_cast<u32x4*>(&Tile[row * LDQ + c8]) = pre[i];
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        Tile[KTILE + (c8 + 2 * e) * LDV + row] = (uint16_t)(pre[i][e] & 0xffffu);
        Tile[KTILE + (c8 + 2 * e + 1) * LDV + row] = (uint16_t)(pre[i][e] >> 16);
      }
    }
  }
  for (int idx = threadIdx.x; idx < (KC - QR) * D; idx += NT) {  // padding keys of the block
    const int r = QR + idx / D, e = idx % D;
    Tile[r * LDQ + e] = 0;
    Tile[KTILE + e * LDV + r] = 0;
  }
  // K rows and V^T rows of a window chunk, from ring slot 0, into the segment's tiles
#define LDR_STASH                                                                        \
  _Pragma("unroll") for (int i = 0; i < PL; ++i) {                                       \
    const int idx_ = (ht + i * ST) % CH;                                                 \
    const int r_ = idx_ / (D / 8), col_ = (idx_ % (D / 8)) * 8;                          \
    *reinterpret_cast<u32x4*>(&Ks[r_ * LDQ + col_]) = wk[0][i];                          \
    *reinterpret_cast<u32x4*>(&Vt[(idx_ >> 2) * LDV + (idx_ & 3) * 8]) = wv[0][i];       \
  }
#define LDR_ADVANCE                                                                      \
  _Pragma("unroll") for (int p = 0; p + 1 < WD; ++p)                                     \
      _Pragma("unroll") for (int i = 0; i < PL; ++i) {                                   \
    wk[p][i] = wk[p + 1][i];                                                             \
    wv[p][i] = wv[p + 1][i];                                                             \
  }                                                                                      \
  LDR_FETCH(WD - 1, max(0, min(nf, cend - 1))) ++nf;
  __syncthreads();

  bf16x8 qf[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) qf[kk] = frag(&Qs[hh][(lane & 15) * LDQ + kk * 32 + (lane >> 4) * 8]);

  f32x4 o[NDT];
#pragma unroll
  for (int n = 0; n < NDT; ++n) o[n] = f32x4{0.f, 0.f, 0.f, 0.f};
  float mrow[4], lrow[4];  // rows (lane / 16) * 4 + v; lrow is this lane's partial sum
#pragma unroll
  for (int v = 0; v < 4; ++v) { mrow[v] = -INFINITY; lrow[v] = 0.f; }
  const float scale = a.inv_sqrt_d;

  // online softmax over a 32-key score tile sc (C layout), valid keys < nvalid
  auto absorb = [&](f32x4 (&sc)[2], int nvalid) {
    float cmax[4];
#pragma unroll
    for (int v = 0; v < 4; ++v) cmax[v] = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int key = kt * 16 + (lane & 15);
        const float s = key < nvalid ? sc[kt][v] * scale : -INFINITY;
        sc[kt][v] = s;
        cmax[v] = fmaxf(cmax[v], s);
      }
    // The reference max of a row moves only when the tile's max exceeds it by
    // more than 8 (or it is still -inf): below that, exp(s - m) stays under
    // e^8, and O and l share the same stale reference, so the result is the
    // same softmax. Rescaling O is rare and skipped by the whole wave.
    bool grow = false;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      cmax[v] = max16(cmax[v]);
      grow |= cmax[v] > mrow[v] + 8.f;
    }
    if (__ballot(grow) != 0) {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const float mnew = cmax[v] > mrow[v] + 8.f ? cmax[v] : mrow[v];
        const float alpha = __expf(mrow[v] - mnew);  // first tile: exp(-inf) = 0
        mrow[v] = mnew;
        lrow[v] *= alpha;
#pragma unroll
        for (int n = 0; n < NDT; ++n) o[n][v] *= alpha;
      }
    }
#pragma unroll
    for (int v = 0; v < 4; ++v)
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        const float p = __expf(sc[kt][v] - mrow[v]);
        sc[kt][v] = p;
        lrow[v] += p;
      }
  };

  // Scores of one 32-key tile (keys kbuf, values vbuf), the online softmax,
  // and O += P V on the same tile.
  auto item = [&](const uint16_t* kbuf, const uint16_t* vbuf, int nvalid) {
    f32x4 sc[2];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      sc[kt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < KS; ++kk)
        sc[kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
            qf[kk], frag(&kbuf[(kt * 16 + (lane & 15)) * LDQ + kk * 32 + (lane >> 4) * 8]),
            sc[kt], 0, 0, 0);
    }
    absorb(sc, nvalid);
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int v = 0; v < 4; ++v)
        Pt[w][((lane >> 4) * 4 + v) * LDV + kt * 16 + (lane & 15)] = f32_to_bf16(sc[kt][v]);
    wave_lds_sync();
    const bf16x8 pf = frag(&Pt[w][(lane & 15) * LDV + (lane >> 4) * 8]);
#pragma unroll
    for (int n = 0; n < NDT; ++n)
      o[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
          pf, frag(&vbuf[(n * 16 + (lane & 15)) * LDV + (lane >> 4) * 8]), o[n], 0, 0, 0);
    wave_lds_sync();
  };

  // ---- the segments walk their items in step: stage, barrier, compute,
  // barrier. Segment 0's first item is the block, staged above.
  for (int it = 0; it < steps; ++it) {
    if (it > 0 || seg != 0) {
      LDR_STASH   // the segment's next chunk (past its end: unused)
      LDR_ADVANCE
      lds_barrier();
    } else {
      lds_barrier();
    }
    if (it < items) {
      const int chunk = cbeg + it - (seg == 0 ? 1 : 0);  // -1: the block
      const int nvalid = chunk < cbeg ? B : chunk_valid(chunk);
      if (nvalid > 0) item(Ks, Vt, nvalid);
    }
    lds_barrier();
  }
#undef LDR_ADVANCE
#undef LDR_STASH
#undef LDR_FETCH

  // ---- summary of the heads (last segment): G rows as keys, M^T (bf16) as
  // values, one more 32-key item with keys R .. 31 masked and their values zero
#pragma unroll
  for (int i = 0; i < GL; ++i) {
    const int idx = threadIdx.x + i * NT;
    if (idx < SG) {
      const int hq_ = idx / (RMAX * D / 8), r = (idx / (D / 8)) % RMAX, col = (idx % (D / 8)) * 8;
      *reinterpret_cast<uint4*>(&Gs[hq_ * RMAX * LDQ + r * LDQ + col]) = greg[i];
    }
  }
#pragma unroll
  for (int i = 0; i < ML; ++i) {  // M^T in bf16: Mt[head][e][r]
    const int idx = threadIdx.x + i * NT;
    if (idx < SM) {
      const int hq_ = idx / (RMAX * D / 4), r = idx % RMAX, col = ((idx / RMAX) % (D / 4)) * 4;
      const uint32_t m4[4] = {mreg[i].x, mreg[i].y, mreg[i].z, mreg[i].w};
#pragma unroll
      for (int k = 0; k < 4; ++k)
        Mt[hq_ * VTILE + (col + k) * LDV + r] = f32_to_bf16(__uint_as_float(m4[k]));
    }
  }
  for (int idx = threadIdx.x; idx < HPW * D * (KC - RMAX) / 8; idx += NT) {  // keys 16..31
    const int hq_ = idx / (D * (KC - RMAX) / 8), rest = idx % (D * (KC - RMAX) / 8);
    *reinterpret_cast<u32x4*>(&Mt[hq_ * VTILE + (rest / 2) * LDV + RMAX + (rest % 2) * 8]) =
        u32x4{0u, 0u, 0u, 0u};
  }
  __syncthreads();
  if (seg == NSEG - 1 && t > 0 && a.use_summary) {
    f32x4 sc[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
#pragma unroll
    for (int kk = 0; kk < KS; ++kk)
      sc[0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
          qf[kk], frag(&Gs[hh * RMAX * LDQ + (lane & 15) * LDQ + kk * 32 + (lane >> 4) * 8]),
          sc[0], 0, 0, 0);
    absorb(sc, a.R);
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int v = 0; v < 4; ++v)
        Pt[w][((lane >> 4) * 4 + v) * LDV + kt * 16 + (lane & 15)] = f32_to_bf16(sc[kt][v]);
    wave_lds_sync();
    const bf16x8 pf = frag(&Pt[w][(lane & 15) * LDV + (lane >> 4) * 8]);
#pragma unroll
    for (int n = 0; n < NDT; ++n)
      o[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
          pf, frag(&Mt[hh * VTILE + (n * 16 + (lane & 15)) * LDV + (lane >> 4) * 8]), o[n], 0, 0, 0);
  }
  __syncthreads();

  // ---- merge: segments 1 .. NSEG - 1 park (O, m, l), segment 0 combines and writes o
  if (seg > 0) {
    const int base = (seg - 1) * HPW + hh;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int q = (lane >> 4) * 4 + v;
      const float l = sum16(lrow[v]);
#pragma unroll
      for (int n = 0; n < NDT; ++n) Xo[(base * QR + q) * D + n * 16 + (lane & 15)] = o[n][v];
      if ((lane & 15) == 0) {
        Xml[(base * QR + q) * 2] = mrow[v];
        Xml[(base * QR + q) * 2 + 1] = l;
      }
    }
  }
  __syncthreads();
  if (seg == 0) {
    uint16_t* out = static_cast<uint16_t*>(a.o);
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int q = (lane >> 4) * 4 + v;
      float m = mrow[v];
#pragma unroll
      for (int sg = 1; sg < NSEG; ++sg) m = fmaxf(m, Xml[(((sg - 1) * HPW + hh) * QR + q) * 2]);
      const float w0 = m == -INFINITY ? 0.f : __expf(mrow[v] - m);
      float den = w0 * sum16(lrow[v]);
      float ws[NSEG];
#pragma unroll
      for (int sg = 1; sg < NSEG; ++sg) {
        const int base = ((sg - 1) * HPW + hh) * QR + q;
        const float ms = Xml[base * 2];
        ws[sg] = ms == -INFINITY ? 0.f : __expf(ms - m);
        den += ws[sg] * Xml[base * 2 + 1];
      }
      const float inv = 1.f / den;
      if (q < B) {
        uint16_t* row = out + ((long)b * B + q) * ((long)a.hq * D) + (long)h * D + (lane & 15);
#pragma unroll
        for (int n = 0; n < NDT; ++n) {
          float acc = w0 * o[n][v];
#pragma unroll
          for (int sg = 1; sg < NSEG; ++sg)
            acc += ws[sg] * Xo[(((sg - 1) * HPW + hh) * QR + q) * D + n * 16 + (lane & 15)];
          row[n * 16] = f32_to_bf16(acc * inv);
        }
      }
    }
  }
}

template <int D>
hipError_t launch_d(const AttnArgs& a, int hkv, int batch, hipStream_t st) {
  // Regions of at least 8 chunks with heads in pairs: two heads per workgroup
  // and four key segments per head (8 waves; 256 workgroups at 8 kv groups x 2
  // head pairs x 16 sequences). Otherwise up to four heads per workgroup and
  // two segments per head.
  const int nwf = a.Wx / KC;
  if (nwf >= 8 && a.rep % 2 == 0) {
    const dim3 grid(hkv * (a.rep / 2), batch);
    hipLaunchKernelGGL((attention_mfma_kernel<D, 2, 4, 2>), grid, dim3(512), 0, st, a);
    return hipGetLastError();
  }
  const int hpw = a.rep < 4 ? a.rep : 4;
  const dim3 grid(hkv * (a.rep / hpw), batch);
  switch (hpw) {
    case 1: hipLaunchKernelGGL((attention_mfma_kernel<D, 1, 2, 4>), grid, dim3(128), 0, st, a); break;
    case 2: hipLaunchKernelGGL((attention_mfma_kernel<D, 2, 2, 4>), grid, dim3(256), 0, st, a); break;
    default: hipLaunchKernelGGL((attention_mfma_kernel<D, 4, 2, 4>), grid, dim3(512), 0, st, a); break;
  }
  return hipGetLastError();
}

}  // namespace

bool attention_mfma_supported(int d, int rep, int B, int R, int W) {   // W: region rows
  return (d == 64 || d == 128) && (rep == 1 || rep == 2 || rep % 4 == 0) && rep <= 64 &&
         B <= QR && R <= 16 && W % (2 * KC) == 0;
}

hipError_t launch_attention_mfma(const AttnArgs& a, int hkv, int batch, hipStream_t st) {
  if (!attention_mfma_supported(a.d, a.rep, a.B, a.R, a.W)) return hipErrorInvalidValue;
  return a.d == 128 ? launch_d<128>(a, hkv, batch, st) : launch_d<64>(a, hkv, batch, st);
}

}  // namespace ldr
