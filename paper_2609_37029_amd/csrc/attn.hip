// Block-view attention on MFMA for bf16 views (Eq. 6; App. A.1; Sec. 2.4).
//
// One workgroup per (kv group g, sequence b, HPW query heads of the group),
// NSEG waves per head, each taking one segment of the key sources under its
// own online softmax: segment 0 the block's own k / v (B rows) and the first
// window chunks, the last
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
// The block's q, k and v are finished in the prologue from the QKV
// projection's fp32 split-K partials: the split sum, the per-head RMSNorm of
// q and k with their gains, and rotate-half RoPE (Sec. 2.4), rounded to bf16
// into LDS. The k / v of a group are finished by each workgroup that reads
// them (rep / HPW of them).
#include "ldr_internal.h"

namespace ldr {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int KC = 32;  // keys per chunk
constexpr int QR = 16;  // query rows per wave (block slots, zero-padded)

__device__ inline bf16x8 frag(const uint16_t* p) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(p));
}
__device__ inline void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

// HPW query heads of one kv group per workgroup (a group with more heads
// spreads over rep / HPW workgroups, each reading the group's window), NSEG
// waves per head: the window chunks are cut into NSEG segments, and every wave
// keeps the online-softmax state of its segment. Segment 0 also takes the
// block's own k / v and the last segment the R summary entries, both before
// the window chunks: their rows are loaded first and reach LDS while the
// window is still arriving. The segments merge their (max, sum, O) in LDS at
// the end. Each segment stages its chunks through one LDS tile pair (K rows,
// V^T rows), two barriers per step.
//
// Loads complete in issue order per wave, so the kernel issues every load of
// the prologue unconditionally (indices clamped, values masked where used):
// summary, block rows, then WD window chunks per segment. Each later wait then
// covers only what the next stage needs. WIN: the views have window or pooled
// rows. PREFETCHED: no segment has more chunks than the WD the prologue loads.
template <int D, int HPW, int NSEG, int WD, bool WIN, bool PREFETCHED, int SPLITS>
__global__ void __launch_bounds__(64 * HPW * NSEG) attention_mfma_kernel(AttnArgs a) {
  constexpr int NT = 64 * HPW * NSEG, ST = 64 * HPW;  // threads, threads per segment
  constexpr int LDQ = D + 8;   // bf16 row of the Q / K tiles (conflict-free 16-row reads)
  constexpr int LDV = KC + 8;  // bf16 row of the V^T / P tiles
  constexpr int NDT = D / 16, KS = D / 32;
  constexpr int CH = KC * D / 8;              // 16-byte pieces of one chunk matrix
  constexpr int PL = (CH + ST - 1) / ST;      // pieces per thread of its segment
  constexpr int RMAX = 16;
  constexpr int KTILE = KC * LDQ, VTILE = D * LDV, SEGT = KTILE + VTILE;
  // LDS (bf16 units): Q rows, the block tile, summary keys G and values M^T,
  // the segments' chunk tiles; after the loop the merge data overlays all of
  // it. P tiles apart.
  constexpr int OQ = 0, OB = OQ + HPW * QR * LDQ, OG = OB + SEGT, OM = OG + HPW * RMAX * LDQ;
  constexpr int OT = OM + HPW * VTILE, AREA = OT + NSEG * SEGT;
  // The summary values M are fp32: M^T goes to the MFMA as bf16 M_hi plus
  // bf16 M_lo = M - M_hi (rows of LDL keys, the R <= 16 entries), so the P.M
  // product keeps M to about 2^-17 relative. The low halves overlay the
  // segments' chunk tiles, which are first staged after the summary item.
  constexpr int LDL = RMAX + 8, OL = OT;
  static_assert(HPW * D * LDL <= NSEG * SEGT, "M_lo fits in the chunk tiles");
  constexpr int MERGE = NSEG * HPW * QR * (D + 2) * 2;
  __shared__ __attribute__((aligned(16))) uint16_t Lds[AREA > MERGE ? AREA : MERGE];
  __shared__ __attribute__((aligned(16))) uint16_t Pt[HPW * NSEG][QR * LDV];
  uint16_t* const Blk = Lds + OB;
  float* const Xo = reinterpret_cast<float*>(Lds);    // [NSEG][HPW][QR][D]
  float* const Xml = Xo + NSEG * HPW * QR * D;        // [NSEG][HPW][QR][2]

  // blockIdx.x = head set * hkv + group: the workgroups that read one group's
  // window are hkv apart in the dispatch order, so with 8 kv groups they land
  // on the same XCD and share its L2
  const int g = blockIdx.x % a.hkv, b = blockIdx.y;
  const int h0 = g * a.rep + (blockIdx.x / a.hkv) * HPW;  // first head of the workgroup
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int seg = w / HPW, hh = w % HPW, h = h0 + hh;
  const int ht = threadIdx.x - seg * ST;  // thread index inside the segment
  uint16_t* const Ks = Lds + OT + seg * SEGT;
  uint16_t* const Vt = Ks + KTILE;
  const int B = a.B;
  const uint8_t* seq = a.arena + (size_t)b * a.stride;
  // window chunks of the segment, assigned over the full region so that the
  // fetches do not wait for the position t (unfilled slots read as zeros and
  // are masked); the launcher keeps every segment nonempty
  const int nwf = a.Wx / KC;
  const int cbeg = seg * nwf / NSEG, cend = (seg + 1) * nwf / NSEG;

  // the position first: its wait then leaves every later load in flight
  const long t = a.pos[b];
  // ---- summary keys G and values M of the workgroup's heads (rows past R: 0).
  // Without the summary the loads read the first 16 bytes of the projection
  // partials instead (unused), so that every path issues the same loads.
  constexpr int SG = HPW * RMAX * D / 8;      // 16-byte pieces of G (bf16)
  constexpr int SM = HPW * RMAX * D / 4;      // 16-byte pieces of M (fp32)
  constexpr int GL = (SG + NT - 1) / NT, ML = (SM + NT - 1) / NT;
  const bool use_sum = a.use_summary != 0;
  uint4 greg[GL], mreg[ML];
  {
    const size_t hrow = (size_t)(a.layer * a.hq + h0) * a.R;  // first row of the workgroup
    const uint16_t* Gg = use_sum ? static_cast<const uint16_t*>(a.G) + hrow * D
                                 : reinterpret_cast<const uint16_t*>(a.part);
    const float* Mg = use_sum ? reinterpret_cast<const float*>(seq + a.m_off) + hrow * D
                              : a.part;
#pragma unroll
    for (int i = 0; i < GL; ++i) {
      const int idx = min(threadIdx.x + i * NT, SG - 1);
      const int hq_ = idx / (RMAX * D / 8), r = min((idx / (D / 8)) % RMAX, a.R - 1);
      const size_t off = ((size_t)hq_ * a.R + r) * D + (idx % (D / 8)) * 8;
      greg[i] = *reinterpret_cast<const uint4*>(Gg + (use_sum ? off : 0));
    }
#pragma unroll
    for (int i = 0; i < ML; ++i) {
      const int idx = min(threadIdx.x + i * NT, SM - 1);
      const int hq_ = idx / (RMAX * D / 4), r = min(idx % RMAX, a.R - 1);
      const size_t off = ((size_t)hq_ * a.R + r) * D + ((idx / RMAX) % (D / 4)) * 4;
      mreg[i] = *reinterpret_cast<const uint4*>(Mg + (use_sum ? off : 0));
    }
  }

  // ---- block rows, finished here from the QKV projection's fp32 split-K
  // partials: q of the workgroup's heads, k and v of the group, for rows
  // min(i, B - 1) of the 16-row tile. A piece is elements e .. e + 7 and
  // e + D/2 .. e + D/2 + 7 (e = 8 x piece) of one (row, head slot) unit, so
  // that it holds whole rotary pairs (rotate-half RoPE); the PPU pieces of a
  // unit sit on consecutive lanes. Units: q heads (slot < HPW), k, v.
  constexpr int HALF = D / 2, PPU = D / 16, NU = (HPW + 2) * QR, NPC = NU * PPU;
  constexpr int FI = (NPC + NT - 1) / NT;     // pieces per thread
  static_assert(64 % PPU == 0, "a unit's pieces in one wave");
  float4 fp[FI][SPLITS][4];                   // partials: e .. + 3, + 4 .. + 7, e + D/2 ..
  u32x4 gq[FI][2];                            // q or k gains of the piece (bf16)
  float4 rc[FI][4];                           // cos, sin of the piece's row (e .. + 7)
  auto piece = [&](int f, int& unit_slot, int& row, int& pc) {
    const int idx = min((int)threadIdx.x + f * NT, NPC - 1);
    const int u = idx / PPU;
    pc = idx % PPU; unit_slot = u / QR; row = u % QR;
  };
#pragma unroll
  for (int f = 0; f < FI; ++f) {
    int us, row, pc;
    piece(f, us, row, pc);
    const int hs = us < HPW ? h0 + us : us == HPW ? a.hq + g : a.hq + a.hkv + g;
    const long m = (long)b * B + min(row, B - 1);
    const float* src = a.part + m * a.qkv_out + (long)hs * D + pc * 8;
#pragma unroll
    for (int sp = 0; sp < SPLITS; ++sp) {
      const float* ps = src + sp * a.split_stride;
      fp[f][sp][0] = *reinterpret_cast<const float4*>(ps);
      fp[f][sp][1] = *reinterpret_cast<const float4*>(ps + 4);
      fp[f][sp][2] = *reinterpret_cast<const float4*>(ps + HALF);
      fp[f][sp][3] = *reinterpret_cast<const float4*>(ps + HALF + 4);
    }
    const uint16_t* gain = static_cast<const uint16_t*>(us < HPW ? a.q_norm : a.k_norm) + pc * 8;
    gq[f][0] = *reinterpret_cast<const u32x4*>(gain);
    gq[f][1] = *reinterpret_cast<const u32x4*>(gain + HALF);
    const float* cs = a.rope + m * HALF + pc * 8;
    const float* sn = cs + (long)a.rows * HALF;
    rc[f][0] = *reinterpret_cast<const float4*>(cs);
    rc[f][1] = *reinterpret_cast<const float4*>(cs + 4);
    rc[f][2] = *reinterpret_cast<const float4*>(sn);
    rc[f][3] = *reinterpret_cast<const float4*>(sn + 4);
  }
  // the window loads stay behind these in issue order, so that finishing the
  // block rows waits for its own loads only (the scheduler does not move
  // loads across this point)
  __builtin_amdgcn_sched_barrier(0);

  // ---- window chunks: ring slot p holds the segment's chunk cbeg + p (the
  // last one repeated for a segment with fewer chunks)
  const size_t gw = (size_t)(a.layer * a.hkv + g) * a.Wx * D;   // window rows, then pooled slots
  const uint16_t* Kw = reinterpret_cast<const uint16_t*>(seq + a.kw) + gw;
  const uint16_t* Vw = reinterpret_cast<const uint16_t*>(seq + a.vw) + gw;
  u32x4 wk[WD][PL], wv[WD][PL];
#define LDR_FETCH(p, c)                                                                  \
  _Pragma("unroll") for (int i = 0; i < PL; ++i) {                                       \
    const int idx_ = (ht + i * ST) % CH;                                                 \
    const int slot_ = (c) * KC + idx_ / (D / 8), col_ = (idx_ % (D / 8)) * 8;            \
    wk[p][i] = *reinterpret_cast<const u32x4*>(Kw + (size_t)slot_ * D + col_);         \
    wv[p][i] = *reinterpret_cast<const u32x4*>(Vw + (size_t)(idx_ >> 2) * a.Wx +        \
                                               (c) * KC + (idx_ & 3) * 8);               \
  }
  if constexpr (WIN) {
#pragma unroll
    for (int p = 0; p < WD; ++p) { LDR_FETCH(p, min(cbeg + p, cend - 1)) }
  }

  // ---- Q, the block tile and the summary tiles into LDS. Finishing a piece:
  // the split sum (in split order), then for q and k the per-head RMSNorm
  // (sum of squares over the unit's lanes) with its gain and the rotation of
  // each pair (e, e + D/2) by the row's angle; rows past B are 0.
#pragma unroll
  for (int f = 0; f < FI; ++f) {
    int us, row, pc;
    piece(f, us, row, pc);
    float x1[8], x2[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      x1[j] = 0.f; x2[j] = 0.f;
#pragma unroll
      for (int sp = 0; sp < SPLITS; ++sp) {
        x1[j] += fp[f][sp][j >> 2][j & 3];
        x2[j] += fp[f][sp][2 + (j >> 2)][j & 3];
      }
    }
    float ss = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) ss += x1[j] * x1[j] + x2[j] * x2[j];
    ss += dpp<0xB1>(ss);                       // the unit's PPU lanes (4 or 8)
    ss += dpp<0x4E>(ss);
    if constexpr (PPU == 8) ss += dpp<0x141>(ss);
    if (us <= HPW) {                           // q or k
      const float inv = rsqrtf(ss / D + a.eps);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const uint32_t w1 = gq[f][0][j >> 1], w2 = gq[f][1][j >> 1];
        const float g1 = bf16_to_f32((uint16_t)(j & 1 ? w1 >> 16 : w1 & 0xffffu));
        const float g2 = bf16_to_f32((uint16_t)(j & 1 ? w2 >> 16 : w2 & 0xffffu));
        const float z1 = x1[j] * inv * g1, z2 = x2[j] * inv * g2;
        const float c = rc[f][j >> 2][j & 3], sn = rc[f][2 + (j >> 2)][j & 3];
        x1[j] = z1 * c - z2 * sn;
        x2[j] = z1 * sn + z2 * c;
      }
    }
    if ((int)threadIdx.x + f * NT >= NPC) continue;
    const bool live = row < B;
    uint32_t h1[4], h2[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      h1[j] = live ? (uint32_t)f32_to_bf16(x1[2 * j]) | ((uint32_t)f32_to_bf16(x1[2 * j + 1]) << 16) : 0u;
      h2[j] = live ? (uint32_t)f32_to_bf16(x2[2 * j]) | ((uint32_t)f32_to_bf16(x2[2 * j + 1]) << 16) : 0u;
    }
    const int c8 = pc * 8;
    if (us < HPW || us == HPW) {
      uint16_t* dst = us < HPW ? &Lds[OQ + us * QR * LDQ + row * LDQ] : &Blk[row * LDQ];
      *reinterpret_cast<u32x4*>(dst + c8) = u32x4{h1[0], h1[1], h1[2], h1[3]};
      *reinterpret_cast<u32x4*>(dst + HALF + c8) = u32x4{h2[0], h2[1], h2[2], h2[3]};
    } else {                                   // v, transposed: V^T[e][row]
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        Blk[KTILE + (c8 + j) * LDV + row] = (uint16_t)(h1[j >> 1] >> (16 * (j & 1)));
        Blk[KTILE + (HALF + c8 + j) * LDV + row] = (uint16_t)(h2[j >> 1] >> (16 * (j & 1)));
      }
    }
  }
  for (int idx = threadIdx.x; idx < (KC - QR) * D; idx += NT) {  // padding keys of the block
    const int r = QR + idx / D, e = idx % D;
    Blk[r * LDQ + e] = 0;
    Blk[KTILE + e * LDV + r] = 0;
  }
#pragma unroll
  for (int i = 0; i < GL; ++i) {
    const int idx = threadIdx.x + i * NT;
    if (idx < SG) {
      const int hq_ = idx / (RMAX * D / 8), r = (idx / (D / 8)) % RMAX, col = (idx % (D / 8)) * 8;
      *reinterpret_cast<uint4*>(&Lds[OG + hq_ * RMAX * LDQ + r * LDQ + col]) =
          use_sum && r < a.R ? greg[i] : make_uint4(0, 0, 0, 0);
    }
  }
#pragma unroll
  for (int i = 0; i < ML; ++i) {  // M^T as bf16 high and low parts: Mt[head][e][r]
    const int idx = threadIdx.x + i * NT;
    if (idx < SM) {
      const int hq_ = idx / (RMAX * D / 4), r = idx % RMAX, col = ((idx / RMAX) % (D / 4)) * 4;
      const bool ok = use_sum && r < a.R;
      uint32_t m4[4] = {mreg[i].x, mreg[i].y, mreg[i].z, mreg[i].w};
      // keeps the conversion here: moved up to the loads, it would wait for them there
      asm volatile("" : "+v"(m4[0]), "+v"(m4[1]), "+v"(m4[2]), "+v"(m4[3]));
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const float m = __uint_as_float(m4[k]);
        const uint16_t hi = f32_to_bf16(m);
        Lds[OM + hq_ * VTILE + (col + k) * LDV + r] = ok ? hi : 0;
        Lds[OL + hq_ * D * LDL + (col + k) * LDL + r] = ok ? f32_to_bf16(m - bf16_to_f32(hi)) : 0;
      }
    }
  }
  for (int idx = threadIdx.x; idx < HPW * D * (KC - RMAX) / 8; idx += NT) {  // keys 16..31
    const int hq_ = idx / (D * (KC - RMAX) / 8), rest = idx % (D * (KC - RMAX) / 8);
    *reinterpret_cast<u32x4*>(&Lds[OM + hq_ * VTILE + (rest / 2) * LDV + RMAX + (rest % 2) * 8]) =
        u32x4{0u, 0u, 0u, 0u};
  }

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
  // window items of a segment: its chunks below nwin
  auto seg_items = [&](int sg) -> int {
    const int c0 = sg * nwf / NSEG, c1 = (sg + 1) * nwf / NSEG;
    return max(0, min(nwin, c1) - c0);
  };
  const int items = seg_items(seg);
  int steps = 0;   // the same on every thread: every wave meets every barrier
#pragma unroll
  for (int sg = 0; sg < NSEG; ++sg) steps = max(steps, seg_items(sg));
  lds_barrier();   // the staged tiles are whole; the window loads stay in flight

  bf16x8 qf[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk)
    qf[kk] = frag(&Lds[OQ + hh * QR * LDQ + (lane & 15) * LDQ + kk * 32 + (lane >> 4) * 8]);

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
  // O += P V for the probabilities of a score tile, through the wave's P tile
  // (vlo: the low parts of the first 16 keys' values, rows of LDL)
  auto pv = [&](f32x4 (&sc)[2], const uint16_t* vbuf, const uint16_t* vlo = nullptr) {
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
    if (vlo) {
      const bool low_keys = (lane >> 4) < 2;   // keys 0 .. 15; keys 16 .. 31 carry 0
#pragma unroll
      for (int n = 0; n < NDT; ++n) {
        const bf16x8 lf = frag(&vlo[(n * 16 + (lane & 15)) * LDL + (low_keys ? (lane >> 4) * 8 : 0)]);
        o[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pf, low_keys ? lf : bf16x8{}, o[n], 0, 0, 0);
      }
    }
    wave_lds_sync();
  };
  // scores of one 32-key tile (keys kbuf, values vbuf), softmax, O += P V
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
    pv(sc, vbuf);
  };

  // ---- first items, on rows already in LDS: the block (segment 0) and the
  // summary (last segment: G rows as keys, M^T as values, keys R .. 31 masked)
  if (seg == 0) item(Blk, Blk + KTILE, B);
  if (seg == NSEG - 1 && t > 0 && use_sum) {
    f32x4 sc[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
#pragma unroll
    for (int kk = 0; kk < KS; ++kk)
      sc[0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
          qf[kk], frag(&Lds[OG + hh * RMAX * LDQ + (lane & 15) * LDQ + kk * 32 + (lane >> 4) * 8]),
          sc[0], 0, 0, 0);
    absorb(sc, a.R);
    pv(sc, Lds + OM + hh * VTILE, Lds + OL + hh * D * LDL);
  }
  lds_barrier();   // every wave is past the summary item: the chunk tiles are free

  // ---- the segments walk their window chunks in step: stage, barrier,
  // compute, barrier
#define LDR_STASH(p)                                                                     \
  _Pragma("unroll") for (int i = 0; i < PL; ++i) {                                       \
    const int idx_ = (ht + i * ST) % CH;                                                 \
    const int r_ = idx_ / (D / 8), col_ = (idx_ % (D / 8)) * 8;                          \
    *reinterpret_cast<u32x4*>(&Ks[r_ * LDQ + col_]) = wk[p][i];                          \
    *reinterpret_cast<u32x4*>(&Vt[(idx_ >> 2) * LDV + (idx_ & 3) * 8]) = wv[p][i];       \
  }
  if constexpr (WIN) {
    if constexpr (PREFETCHED) {
#pragma unroll
      for (int it = 0; it < WD; ++it) {
        if (it < steps) {
          LDR_STASH(it)
          lds_barrier();
          if (it < items) item(Ks, Vt, chunk_valid(cbeg + it));
          lds_barrier();
        }
      }
    } else {
      for (int it0 = 0; it0 < steps; it0 += WD) {
#pragma unroll
        for (int j = 0; j < WD; ++j) {
          const int it = it0 + j;
          if (it < steps) {
            LDR_STASH(j)
            // refill the slot (every step issues the same loads, so that the
            // waits stay exact; past the segment's end it repeats its last chunk)
            LDR_FETCH(j, min(cbeg + it + WD, cend - 1))
            lds_barrier();
            if (it < items) item(Ks, Vt, chunk_valid(cbeg + it));
            lds_barrier();
          }
        }
      }
    }
  }
#undef LDR_STASH
#undef LDR_FETCH

  // ---- merge: every wave parks (O, m, l) of its segment; then each wave
  // combines the D / NSEG columns [seg * D / NSEG, ...) of its head over the
  // segments and writes them
  lds_barrier();   // the first items' LDS reads are done (no loop step may have run)
  {
    const int base = (seg * HPW + hh) * QR;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int q = (lane >> 4) * 4 + v;
      const float l = sum16(lrow[v]);
#pragma unroll
      for (int n = 0; n < NDT; ++n) Xo[(base + q) * D + n * 16 + (lane & 15)] = o[n][v];
      if ((lane & 15) == 0) {
        Xml[(base + q) * 2] = mrow[v];
        Xml[(base + q) * 2 + 1] = l;
      }
    }
  }
  lds_barrier();
  constexpr int CW = D / NSEG, CPL = CW / 4;   // columns per wave, per lane (4 lanes a row)
  static_assert(CPL % 4 == 0, "whole 4-column groups per lane");
  {
    const int q = lane >> 2, c0 = seg * CW + (lane & 3) * CPL;
    float m = -INFINITY;
#pragma unroll
    for (int sg = 0; sg < NSEG; ++sg) m = fmaxf(m, Xml[((sg * HPW + hh) * QR + q) * 2]);
    float ws[NSEG], den = 0.f;
#pragma unroll
    for (int sg = 0; sg < NSEG; ++sg) {
      const int r = (sg * HPW + hh) * QR + q;
      const float ms = Xml[r * 2];
      ws[sg] = ms == -INFINITY ? 0.f : __expf(ms - m);
      den += ws[sg] * Xml[r * 2 + 1];
    }
    const float inv = 1.f / den;
    float acc[CPL];
#pragma unroll
    for (int c = 0; c < CPL; ++c) acc[c] = 0.f;
#pragma unroll
    for (int sg = 0; sg < NSEG; ++sg) {
      const float* src = Xo + ((sg * HPW + hh) * QR + q) * D + c0;
#pragma unroll
      for (int c = 0; c < CPL; c += 4) {
        const float4 x = *reinterpret_cast<const float4*>(src + c);
        acc[c] += ws[sg] * x.x;
        acc[c + 1] += ws[sg] * x.y;
        acc[c + 2] += ws[sg] * x.z;
        acc[c + 3] += ws[sg] * x.w;
      }
    }
    if (q < B) {
      uint32_t pk[CPL / 2];
#pragma unroll
      for (int c = 0; c < CPL / 2; ++c)
        pk[c] = (uint32_t)f32_to_bf16(acc[2 * c] * inv) |
                ((uint32_t)f32_to_bf16(acc[2 * c + 1] * inv) << 16);
      const long m = (long)b * B + q, K = (long)a.hq * D;
      uint16_t* o = static_cast<uint16_t*>(a.o);
#pragma unroll
      for (int c = 0; c < CPL / 2; c += 2) {
        // 4 columns k .. k + 3 (k a multiple of 4): 8 bytes of one row, inside
        // one 16-byte chunk of the fragment layout
        const long k = (long)h * D + c0 + 2 * c;
        const long off = a.o_frag ? ((m >> 4) * (K >> 5) + (k >> 5)) * 512 +
                                        ((k >> 3) & 3) * 128 + (m & 15) * 8 + (k & 7)
                                  : m * K + k;
        *reinterpret_cast<uint2*>(o + off) = make_uint2(pk[c], pk[c + 1]);
      }
    }
  }
}

template <int D, int HPW, int NSEG, int WD, int SPLITS>
void launch_cfg(const AttnArgs& a, dim3 grid, hipStream_t st) {
  const int nwf = a.Wx / KC;
  const bool pre = (nwf + NSEG - 1) / NSEG <= WD;   // every segment's chunks fit in the ring
  if (a.Wx == 0)
    hipLaunchKernelGGL((attention_mfma_kernel<D, HPW, NSEG, WD, false, true, SPLITS>), grid,
                       dim3(64 * HPW * NSEG), 0, st, a);
  else if (pre)
    hipLaunchKernelGGL((attention_mfma_kernel<D, HPW, NSEG, WD, true, true, SPLITS>), grid,
                       dim3(64 * HPW * NSEG), 0, st, a);
  else
    hipLaunchKernelGGL((attention_mfma_kernel<D, HPW, NSEG, WD, true, false, SPLITS>), grid,
                       dim3(64 * HPW * NSEG), 0, st, a);
}

template <int D, int HPW, int NSEG, int WD>
void launch_splits(const AttnArgs& a, dim3 grid, hipStream_t st) {
  switch (a.splits) {
    case 1: launch_cfg<D, HPW, NSEG, WD, 1>(a, grid, st); break;
    case 2: launch_cfg<D, HPW, NSEG, WD, 2>(a, grid, st); break;
    default: launch_cfg<D, HPW, NSEG, WD, 4>(a, grid, st); break;
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
    launch_splits<D, 2, 4, 2>(a, dim3(hkv * (a.rep / 2), batch), st);
    return hipGetLastError();
  }
  const int hpw = a.rep < 4 ? a.rep : 4;
  const dim3 grid(hkv * (a.rep / hpw), batch);
  switch (hpw) {
    case 1: launch_splits<D, 1, 2, 4>(a, grid, st); break;
    case 2: launch_splits<D, 2, 2, 4>(a, grid, st); break;
    default: launch_splits<D, 4, 2, 4>(a, grid, st); break;
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
  if (a.splits != 1 && a.splits != 2 && a.splits != 4) return hipErrorInvalidValue;
  return a.d == 128 ? launch_d<128>(a, hkv, batch, st) : launch_d<64>(a, hkv, batch, st);
}

}  // namespace ldr
