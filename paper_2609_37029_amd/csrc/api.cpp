// Host side of the C ABI: configuration checks, the per-sequence arena
// layout, the workspace plan of one draft step, argument validation and the
// launch sequence. Every step of the drafting computation runs in the HIP
// kernels of views.hip, gemm.hip, draft.hip, attn.hip, sample.hip and
// verify.hip.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstring>
#include <new>

#include "ldr_internal.h"

namespace ldr {
int views_dims_per_thread(const Shape& s);

bool make_shape(const ldr_config* c, Shape* s) {
  if (!c) return false;
  if (c->hidden <= 0 || c->hidden % 64) return false;
  if (c->n_q_heads <= 0 || c->n_kv_heads <= 0 || c->n_q_heads % c->n_kv_heads) return false;
  if (c->head_dim != 64 && c->head_dim != 128) return false;
  if (c->mlp <= 0 || c->mlp % 64) return false;
  if (c->vocab <= 0) return false;
  if (c->n_layers <= 0 || c->n_feat_layers <= 0) return false;
  if (c->block < 1 || c->block > 16) return false;
  if (c->window < 1) return false;
  if (c->pool_slots < 0 || (c->pool_slots > 0 && (c->pool_slots % 32 || c->pool_stride[0] < 1 ||
                                                   c->pool_stride[1] < 1)))
    return false;
  if (c->pool_slots == 0 && c->summary < 1) return false;
  if (c->dtype != LDR_F32 && c->dtype != LDR_BF16) return false;
  if (!(c->rms_eps > 0.f) || !(c->rope_theta > 0.f) || !(c->ntk_alpha > 0.f)) return false;
  const int all = LDR_DROP_WINDOW | LDR_DROP_SUMMARY | LDR_DROP_BOUNDARY;
  if ((c->drop_views & ~all) || c->drop_views == all) return false;   // at least one view
  s->hidden = c->hidden; s->hq = c->n_q_heads; s->hkv = c->n_kv_heads; s->d = c->head_dim;
  s->mlp = c->mlp; s->vocab = c->vocab; s->D = c->n_layers; s->Lb = c->n_feat_layers;
  s->B = c->block; s->W = c->window; s->R = c->summary; s->dtype = c->dtype;
  s->rep = s->hq / s->hkv;
  s->qkv_out = (s->hq + 2 * s->hkv) * s->d;
  s->eps = c->rms_eps;
  s->rope_base = (double)c->rope_theta *
                 std::pow((double)c->ntk_alpha, (double)s->d / (double)(s->d - 2));
  s->el = c->dtype == LDR_BF16 ? 2 : 4;
  s->keep_win = !(c->drop_views & LDR_DROP_WINDOW);
  s->keep_sum = !(c->drop_views & LDR_DROP_SUMMARY);
  s->keep_bnd = !(c->drop_views & LDR_DROP_BOUNDARY);
  s->P = s->keep_sum ? c->pool_slots : 0;
  s->S0 = c->pool_stride[0]; s->S1 = c->pool_stride[1];
  s->learned = s->keep_sum && c->pool_slots == 0;
  if (!s->learned) s->R = 0;   // no learned summary queries
  s->Wr = s->keep_win ? s->W : 0;
  s->Wx = s->Wr + 2 * s->P;
  if (views_dims_per_thread(*s) == 0 || !norm_hidden_supported(s->hidden)) return false;
  if (s->dtype == LDR_BF16) {
    if (!attention_mfma_supported(s->d, s->rep, s->B, s->R, s->Wx)) return false;
    // GEMM K dimensions in whole pairs of 64-element steps of the bf16 main loop
    if (s->hidden % 128 || s->mlp % 128 || (s->hq * s->d) % 128) return false;
  }
  return true;
}

Layout make_layout(const Shape& s) {
  Layout L;
  // a dropped view has zero bytes (its offset is that of the next region);
  // the pooled banks' slot means follow the window rows of each (layer, group)
  const size_t win = (size_t)s.D * s.hkv * s.Wx * s.d * s.el;
  const size_t sum = s.learned ? (size_t)s.D * s.hq * s.R : 0;
  L.kw = 0;
  L.vw = align_up(L.kw + win);
  L.m = align_up(L.vw + win);
  L.eta = align_up(L.m + sum * s.d * 4);
  L.h = align_up(L.eta + sum * 4);
  L.ps = align_up(L.h + (s.keep_bnd ? (size_t)s.Lb * s.hidden * s.el : 0));
  L.bytes = L.ps + (s.P ? (size_t)s.D * s.hkv * 2 * 2 * s.d * 4 : 0);
  L.stride = align_up(L.bytes);
  return L;
}

// Workspace regions of one draft step for `batch` sequences.
struct WsPlan {
  size_t part, x, nrm, qkvb, o, act, rope, nrmt, nrmf, bytes;
  GemmPlan fc, qkv, wo, gu, down, lm;
};

static WsPlan plan_ws(const Shape& s, int batch) {
  WsPlan w;
  const int M = batch * s.B;
  w.fc = plan_gemm(s.dtype, batch, s.hidden, s.Lb * s.hidden, true);
  // at most 4 QKV splits in bf16: the attention kernel holds them all in registers
  w.qkv = plan_gemm(s.dtype, M, s.qkv_out, s.hidden, true, false, true,
                    s.dtype == LDR_BF16 ? 4 : 8);
  w.wo = plan_gemm(s.dtype, M, s.hidden, s.hq * s.d, true, false, true);
  w.gu = plan_gemm(s.dtype, M, 2 * s.mlp, s.hidden, false, true);   // SwiGLU epilogue: no split
  // the down projection reads the SwiGLU rows in the fragment layout when the
  // SwiGLU GEMM (itself on the fragment layout) can write them so
  w.down = plan_gemm(s.dtype, M, s.hidden, s.mlp, true, false, gemm_plan_frag(w.gu));
  w.lm = plan_gemm(s.dtype, M, s.vocab, s.hidden, false);     // writes the logits directly
  size_t part = (size_t)w.fc.splits * batch * s.hidden;
  part = part > (size_t)w.qkv.splits * M * s.qkv_out ? part : (size_t)w.qkv.splits * M * s.qkv_out;
  part = part > (size_t)w.wo.splits * M * s.hidden ? part : (size_t)w.wo.splits * M * s.hidden;
  part = part > (size_t)w.down.splits * M * s.hidden ? part : (size_t)w.down.splits * M * s.hidden;
  size_t off = 0;
  w.part = off; off = align_up(off + part * 4);
  w.x = off; off = align_up(off + (size_t)M * s.hidden * 4);
  w.nrm = off; off = align_up(off + (size_t)M * s.hidden * s.el);
  // finished q / k / v rows (fp32 models; the bf16 attention finishes its own)
  w.qkvb = off; off = align_up(off + (s.dtype == LDR_BF16 ? 0 : (size_t)M * s.qkv_out * s.el));
  // attention output and SwiGLU rows padded to 16 for the fragment layout
  const size_t Mp = (size_t)(M + 15) / 16 * 16;
  w.o = off; off = align_up(off + Mp * s.hq * s.d * s.el);
  w.act = off; off = align_up(off + Mp * s.mlp * s.el);
  w.rope = off; off = align_up(off + (size_t)2 * M * (s.d / 2) * 4);
  // final normalised rows in the tiled layout, for a tiled vocabulary head
  w.nrmt = off; off = align_up(off + (s.dtype == LDR_BF16 ? tiled_elems(M, s.hidden) * 2 : 0));
  // the QKV and SwiGLU GEMMs' rows in the fragment layout (rows padded to 16)
  w.nrmf = off;
  off = align_up(off + (gemm_plan_frag(w.gu) || gemm_plan_frag(w.qkv)
                            ? (size_t)(M + 15) / 16 * 16 * s.hidden * 2 : 0));
  w.bytes = off;
  return w;
}

static bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

}  // namespace ldr

using namespace ldr;

struct ldr_views {
  ldr_config cfg;
  Shape s;
  Layout L;
  int batch;
  uint8_t* arena;
  int64_t* pos;
  const void* G;
  int32_t* status;  // device, 256 bytes: the sticky flags, and at word
                    // kCommitCounter the update's commit counter
};

extern "C" {

int ldr_config_check(const ldr_config* cfg) {
  Shape s;
  return make_shape(cfg, &s) ? LDR_OK : LDR_EINVAL;
}

size_t ldr_views_state_bytes(const ldr_config* cfg) {
  Shape s;
  if (!make_shape(cfg, &s)) return 0;
  return make_layout(s).bytes;
}

size_t ldr_views_stride_bytes(const ldr_config* cfg) {
  Shape s;
  if (!make_shape(cfg, &s)) return 0;
  return make_layout(s).stride;
}

int ldr_views_layout(const ldr_config* cfg, size_t offsets[5]) {
  Shape s;
  if (!offsets || !make_shape(cfg, &s)) return LDR_EINVAL;
  const Layout L = make_layout(s);
  offsets[0] = L.kw; offsets[1] = L.vw; offsets[2] = L.m; offsets[3] = L.eta; offsets[4] = L.h;
  return LDR_OK;
}

size_t ldr_tiled_bytes(int32_t rows, int32_t cols) {
  if (rows <= 0 || cols <= 0 || cols % 32) return 0;
  return tiled_elems(rows, cols) * 2;
}

int ldr_tile_matrix(const void* src, int32_t rows, int32_t cols, int64_t ld, void* dst,
                    size_t dst_bytes, void* stream) {
  if (!src || !dst || rows <= 0 || cols <= 0 || cols % 32 || ld < cols || ld % 8 ||
      !aligned(src, 16) || !aligned(dst, 16) || dst_bytes < ldr_tiled_bytes(rows, cols))
    return LDR_EINVAL;
  return launch_tile_matrix(src, ld, rows, cols, dst, static_cast<hipStream_t>(stream)) ==
                 hipSuccess
             ? LDR_OK
             : LDR_EHIP;
}

size_t ldr_workspace_bytes(const ldr_config* cfg, int32_t batch) {
  Shape s;
  if (batch <= 0 || !make_shape(cfg, &s)) return 0;
  return plan_ws(s, batch).bytes;
}

const char* ldr_strerror(int status) {
  switch (status) {
    case LDR_OK: return "ok";
    case LDR_EINVAL: return "invalid argument";
    case LDR_ERANGE: return "row count out of range";
    case LDR_EHIP: return "HIP runtime error";
    case LDR_ENOMEM: return "out of memory";
    case LDR_ESCRATCH: return "request exceeds the static scratch of the allocation-free call";
    default: return "unknown status";
  }
}

static int views_update_impl(ldr_views* v, const int32_t* n_new, int32_t max_new,
                             const void* K_new, const void* V_new, const void* h_new,
                             hipStream_t st) {
  if (!v || !n_new || max_new < 0) return LDR_EINVAL;
  if (max_new > 0 && (!K_new || !V_new || !aligned(K_new, 16) || !aligned(V_new, 16)))
    return LDR_EINVAL;
  if (v->s.keep_bnd && (!h_new || !aligned(h_new, 16))) return LDR_EINVAL;
  // the last launch that reads t commits from its last workgroup
  int32_t* done = v->status + kCommitCounter;
  if (max_new > 0) {
    if (launch_views_update(v->s, v->L, v->batch, v->arena, v->pos, v->G, n_new, max_new, K_new,
                            V_new, h_new, st, v->status, v->s.P ? nullptr : done) != hipSuccess)
      return LDR_EHIP;
    if (v->s.P && launch_views_pool(v->s, v->L, v->batch, v->arena, v->pos, n_new, max_new,
                                    K_new, V_new, st, v->status, done) != hipSuccess)
      return LDR_EHIP;
    return LDR_OK;
  }
  if (launch_views_commit(v->batch, v->pos, n_new, max_new, v->status, st) != hipSuccess)
    return LDR_EHIP;
  return LDR_OK;
}

int ldr_views_init(ldr_views** out, const ldr_config* cfg, int32_t batch, void* arena,
                   int64_t* pos, const void* G, const int32_t* n_prefix, int32_t max_prefix,
                   const void* K_prefix, const void* V_prefix, const void* h_boundary,
                   void* stream) {
  if (!out) return LDR_EINVAL;
  *out = nullptr;
  Shape s;
  if (!make_shape(cfg, &s) || batch <= 0 || !arena || !pos) return LDR_EINVAL;
  if (s.learned && (!G || !aligned(G, 16))) return LDR_EINVAL;   // G: the summary's queries
  if (!aligned(arena, kAlign) || !aligned(pos, 8)) return LDR_EINVAL;
  if (max_prefix < 0 || (max_prefix > 0 && !n_prefix)) return LDR_EINVAL;
  ldr_views* v = new (std::nothrow) ldr_views;
  if (!v) return LDR_ENOMEM;
  v->cfg = *cfg; v->s = s; v->L = make_layout(s); v->batch = batch;
  v->arena = static_cast<uint8_t*>(arena); v->pos = pos; v->G = G; v->status = nullptr;
  if (hipMalloc(reinterpret_cast<void**>(&v->status), 256) != hipSuccess) {
    delete v;
    return LDR_ENOMEM;
  }
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (hipMemsetAsync(v->status, 0, 256, st) != hipSuccess ||
      launch_views_reset(s, v->L, batch, arena, pos, st) != hipSuccess) {
    ldr_views_destroy(v);
    return LDR_EHIP;
  }
  if (max_prefix > 0) {
    const int rc = views_update_impl(v, n_prefix, max_prefix, K_prefix, V_prefix, h_boundary, st);
    if (rc != LDR_OK) {
      hipStreamSynchronize(st);
      ldr_views_destroy(v);
      return rc;
    }
  }
  *out = v;
  return LDR_OK;
}

int ldr_views_update(ldr_views* v, const int32_t* n_new, int32_t max_new, const void* K_new,
                     const void* V_new, const void* h_new, void* stream) {
  return views_update_impl(v, n_new, max_new, K_new, V_new, h_new,
                           static_cast<hipStream_t>(stream));
}

int ldr_views_status(ldr_views* v, int clear, void* stream) {
  if (!v) return LDR_EINVAL;
  hipStream_t st = static_cast<hipStream_t>(stream);
  int32_t flag = 0;
  if (hipMemcpyAsync(&flag, v->status, sizeof(flag), hipMemcpyDeviceToHost, st) != hipSuccess ||
      hipStreamSynchronize(st) != hipSuccess)
    return LDR_EHIP;
  if (clear && flag) {
    if (hipMemsetAsync(v->status, 0, sizeof(int32_t), st) != hipSuccess ||
        hipStreamSynchronize(st) != hipSuccess)
      return LDR_EHIP;
  }
  if (flag & kFlagRange) return LDR_ERANGE;
  return flag ? LDR_EINVAL : LDR_OK;
}

void ldr_views_destroy(ldr_views* v) {
  if (!v) return;
  if (v->status) hipFree(v->status);
  delete v;
}

static bool weights_ok(const Shape& s, const ldr_weights* w) {
  if (!w || !w->layers) return false;
  const void* top[] = {w->embed, w->mask_emb, w->pos_emb, w->final_norm, w->lm_head};
  for (const void* p : top)
    if (!p || !aligned(p, 16)) return false;
  if (s.keep_bnd)   // the boundary fusion exists only with the boundary view
    for (const void* p : {w->fc_w, w->fc_norm})
      if (!p || !aligned(p, 16)) return false;
  for (int j = 0; j < s.D; ++j) {
    const ldr_layer_weights& L = w->layers[j];
    const void* ps[] = {L.in_norm, L.wqkv, L.q_norm, L.k_norm, L.wo, L.post_norm, L.w_gate_up,
                        L.w_down};
    for (const void* p : ps)
      if (!p || !aligned(p, 16)) return false;
  }
  return true;
}

}  // extern "C"

// The launch sequence of one draft step. `emit(kind, launch)` is called once
// per kernel in order; `launch` performs it. Shared by the kernel-kind query
// and the step itself so the two cannot disagree.
template <typename Emit>
static int draft_sequence(const Shape& s, int D, Emit&& emit) {
  int rc = s.keep_bnd ? emit(LDR_LAUNCH_FC_GEMM, 0) : (int)LDR_OK;   // no boundary: c = 0
  if (rc == LDR_OK) rc = emit(LDR_LAUNCH_SLOT_INIT, 0);
  for (int j = 0; j < D && rc == LDR_OK; ++j) {
    // bf16: the attention kernel finishes q, k and v itself
    const int kinds[] = {LDR_LAUNCH_QKV_GEMM, LDR_LAUNCH_QKV_FINISH, LDR_LAUNCH_ATTENTION,
                         LDR_LAUNCH_O_GEMM,
                         LDR_LAUNCH_POST_NORM, LDR_LAUNCH_GATE_UP_GEMM, LDR_LAUNCH_DOWN_GEMM,
                         LDR_LAUNCH_NEXT_NORM};
    for (int k : kinds)
      if (rc == LDR_OK && !(k == LDR_LAUNCH_QKV_FINISH && s.dtype == LDR_BF16)) rc = emit(k, j);
  }
  if (rc == LDR_OK) rc = emit(LDR_LAUNCH_LM_HEAD, 0);
  return rc;
}

extern "C" int32_t ldr_draft_step_launches(const ldr_config* cfg, int32_t* kinds,
                                           int32_t max_kinds) {
  Shape s;
  if (!make_shape(cfg, &s)) return LDR_EINVAL;
  int32_t n = 0;
  draft_sequence(s, s.D, [&](int kind, int) {
    if (kinds && n < max_kinds) kinds[n] = kind;
    ++n;
    return (int)LDR_OK;
  });
  return n;
}

// Sampling fused into the vocabulary head (tiled head only). T = 0: the
// outputs and the argmax partials' workspace; logits may then be NULL (not
// written). T > 0: the chunk log-masses go to the sampler's workspace `parts`
// (rows of ldL floats) beside the logits, for the chunk draw that follows.
struct FusedSample {
  int32_t* tokens; float* lse; float* logq;
  void* parts;
  float T; int ldL;
};

static int draft_step_impl(const ldr_views* v, const ldr_weights* w, const int32_t* anchor,
                           float* logits, void* workspace, size_t workspace_bytes,
                           void* const* events, int32_t n_events, hipStream_t st,
                           const FusedSample* fs = nullptr) {
  if (!v || !anchor || !workspace || (!logits && !fs)) return LDR_EINVAL;
  const Shape& s = v->s;
  if (!weights_ok(s, w) || !aligned(workspace, kAlign) || (logits && !aligned(logits, 16)))
    return LDR_EINVAL;
  if (events && n_events != ldr_draft_step_launches(&v->cfg, nullptr, 0) + 1) return LDR_EINVAL;
  const int batch = v->batch, M = batch * s.B;
  const WsPlan ws = plan_ws(s, batch);
  if (workspace_bytes < ws.bytes) return LDR_EINVAL;
  if (w->lm_head_tiled && (s.dtype != LDR_BF16 || !aligned(w->lm_head_tiled, 16) ||
                           !gemm_tiled_supported(M, s.vocab, s.hidden)))
    return LDR_EINVAL;
  // The tiled head computes 256-row tiles: below 65 rows the row-major head's
  // 16- to 64-row tiles stream the same weights with less MFMA work.
  const bool tiled_head = w->lm_head_tiled != nullptr && M > 64;
  uint8_t* base = static_cast<uint8_t*>(workspace);
  DraftPtrs p;
  p.arena = v->arena; p.pos = v->pos; p.G = v->G; p.status = v->status;
  p.part = reinterpret_cast<float*>(base + ws.part);
  p.x = reinterpret_cast<float*>(base + ws.x);
  p.nrm = base + ws.nrm; p.qkv = base + ws.qkvb; p.o = base + ws.o; p.act = base + ws.act;
  p.rope = reinterpret_cast<float*>(base + ws.rope);

  int li = 0;
  auto mark = [&](int i) -> bool {
    return !events || !events[i] ||
           hipEventRecord(static_cast<hipEvent_t>(events[i]), st) == hipSuccess;
  };
  auto run = [&](int kind, int j) -> int {
    if (!mark(li)) return LDR_EHIP;
    GemmArgs g;
    g.mlp = 0;
    hipError_t e = hipSuccess;
    const ldr_layer_weights& L = w->layers[j];
    switch (kind) {
      case LDR_LAUNCH_FC_GEMM:  // boundary fusion over the stored boundary states
        g.A = v->arena + v->L.h; g.lda = (long)(v->L.stride / s.el);
        g.W = w->fc_w; g.ldw = (long)s.Lb * s.hidden; g.out = p.part; g.ldo = s.hidden;
        g.split_stride = (long)batch * s.hidden; g.M = batch; g.N = s.hidden;
        g.K = s.Lb * s.hidden; g.splits = ws.fc.splits;
        e = launch_gemm(s.dtype, EPI_STORE, ws.fc, g, st);
        break;
      case LDR_LAUNCH_SLOT_INIT:
        e = launch_slot_init(s, batch, p, ws.fc.splits, w, anchor, st,
                             gemm_plan_frag(ws.qkv) ? base + ws.nrmf : nullptr);
        break;
      case LDR_LAUNCH_QKV_GEMM:
        g.A = gemm_plan_frag(ws.qkv) ? static_cast<const void*>(base + ws.nrmf) : p.nrm;
        g.lda = s.hidden; g.W = L.wqkv; g.ldw = s.hidden; g.out = p.part;
        g.ldo = s.qkv_out; g.split_stride = (long)M * s.qkv_out; g.M = M; g.N = s.qkv_out;
        g.K = s.hidden; g.splits = ws.qkv.splits;
        e = launch_gemm(s.dtype, EPI_STORE, ws.qkv, g, st);
        break;
      case LDR_LAUNCH_QKV_FINISH:
        e = launch_qkv_finish(s, M, p, ws.qkv.splits, &L, st);
        break;
      case LDR_LAUNCH_ATTENTION:
        e = launch_attention(s, v->L, batch, p, j, &L, ws.qkv.splits, st, gemm_plan_frag(ws.wo));
        break;
      case LDR_LAUNCH_O_GEMM:
        g.A = p.o; g.lda = (long)s.hq * s.d; g.W = L.wo; g.ldw = (long)s.hq * s.d;
        g.out = p.part; g.ldo = s.hidden; g.split_stride = (long)M * s.hidden; g.M = M;
        g.N = s.hidden; g.K = s.hq * s.d; g.splits = ws.wo.splits;
        e = launch_gemm(s.dtype, EPI_STORE, ws.wo, g, st);
        break;
      case LDR_LAUNCH_POST_NORM:
        e = gemm_plan_frag(ws.gu)
                ? launch_resid_norm(s, M, p, ws.wo.splits, L.post_norm, st, base + ws.nrmf,
                                    NRM_FRAG)
                : launch_resid_norm(s, M, p, ws.wo.splits, L.post_norm, st);
        break;
      case LDR_LAUNCH_GATE_UP_GEMM:
        g.A = gemm_plan_frag(ws.gu) ? static_cast<const void*>(base + ws.nrmf) : p.nrm;
        g.lda = s.hidden; g.W = L.w_gate_up; g.ldw = s.hidden; g.out = p.act;
        g.ldo = s.mlp; g.split_stride = 0; g.M = M; g.N = 2 * s.mlp; g.K = s.hidden;
        g.splits = 1; g.mlp = s.mlp; g.out_frag = gemm_plan_frag(ws.down);
        e = launch_gemm(s.dtype, EPI_SWIGLU, ws.gu, g, st);
        break;
      case LDR_LAUNCH_DOWN_GEMM:
        g.A = p.act; g.lda = s.mlp; g.W = L.w_down; g.ldw = s.mlp; g.out = p.part;
        g.ldo = s.hidden; g.split_stride = (long)M * s.hidden; g.M = M; g.N = s.hidden;
        g.K = s.mlp; g.splits = ws.down.splits;
        e = launch_gemm(s.dtype, EPI_STORE, ws.down, g, st);
        break;
      case LDR_LAUNCH_NEXT_NORM:
        if (j + 1 < s.D)   // the next layer's QKV input
          e = gemm_plan_frag(ws.qkv)
                  ? launch_resid_norm(s, M, p, ws.down.splits, w->layers[j + 1].in_norm, st,
                                      base + ws.nrmf, NRM_FRAG)
                  : launch_resid_norm(s, M, p, ws.down.splits, w->layers[j + 1].in_norm, st);
        else               // the vocabulary head's input
          e = launch_resid_norm(s, M, p, ws.down.splits, w->final_norm, st,
                                tiled_head ? base + ws.nrmt : nullptr);
        break;
      case LDR_LAUNCH_LM_HEAD:
        g.lda = s.hidden; g.ldw = s.hidden; g.out = logits; g.ldo = s.vocab;
        g.split_stride = 0; g.M = M; g.N = s.vocab; g.K = s.hidden; g.splits = 1;
        if (tiled_head && fs && fs->T > 0.f) {
          g.A = base + ws.nrmt; g.W = w->lm_head_tiled;
          HeadSampleArgs hs{};
          hs.L = static_cast<float*>(fs->parts); hs.ldL = fs->ldL; hs.T = fs->T;
          e = launch_gemm_tiled_chunks(g, hs, st);
        } else if (tiled_head && fs) {
          g.A = base + ws.nrmt; g.W = w->lm_head_tiled;
          HeadSampleArgs hs{};
          hs.parts = fs->parts; hs.store_logits = logits != nullptr;
          e = launch_gemm_tiled_argmax(g, hs, fs->tokens, fs->lse, fs->logq, st);
        } else if (tiled_head) {
          g.A = base + ws.nrmt; g.W = w->lm_head_tiled;
          e = launch_gemm_tiled(g, st);
        } else {
          g.A = p.nrm; g.W = w->lm_head;
          e = launch_gemm(s.dtype, EPI_LOGITS, ws.lm, g, st);
        }
        break;
      default:
        return LDR_EINVAL;
    }
    ++li;
    return e == hipSuccess ? (int)LDR_OK : (int)LDR_EHIP;
  };
  int rc = draft_sequence(s, s.D, run);
  if (rc == LDR_OK && !mark(li)) rc = LDR_EHIP;
  return rc;
}

extern "C" {

int ldr_draft_step(const ldr_views* v, const ldr_weights* w, const int32_t* anchor,
                   float* logits, void* workspace, size_t workspace_bytes, void* stream) {
  return draft_step_impl(v, w, anchor, logits, workspace, workspace_bytes, nullptr, 0,
                         static_cast<hipStream_t>(stream));
}

size_t ldr_draft_step_sample_workspace_bytes(const ldr_config* cfg, int32_t batch) {
  Shape s;
  if (!make_shape(cfg, &s) || batch <= 0) return 0;
  const int rows = batch * s.B;
  const size_t draft = plan_ws(s, batch).bytes;
  const size_t parts = head_sample_part_bytes(rows, s.vocab);
  const size_t samp = ldr_sample_workspace_bytes(rows, s.vocab);
  return align_up(draft) + align_up(parts > samp ? parts : samp);
}

int ldr_draft_step_sample(const ldr_views* v, const ldr_weights* w, const int32_t* anchor,
                          float* logits, float temperature, uint64_t seed, uint64_t step,
                          int32_t* tokens, float* lse, float* logq, void* workspace,
                          size_t workspace_bytes, void* stream) {
  if (!v || !w || !tokens || !lse || !logq || !workspace) return LDR_EINVAL;
  if (!(temperature >= 0.f) || std::isinf(temperature)) return LDR_EINVAL;
  const Shape& s = v->s;
  const int rows = v->batch * s.B;
  if (workspace_bytes < ldr_draft_step_sample_workspace_bytes(&v->cfg, v->batch) ||
      !aligned(workspace, kAlign))
    return LDR_EINVAL;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const size_t draft = align_up(plan_ws(s, v->batch).bytes);
  uint8_t* extra = static_cast<uint8_t*>(workspace) + draft;
  // greedy steps fuse the argmax into the head, which needs its tiled copy
  // and runs above 64 rows
  if (temperature == 0.f && w->lm_head_tiled && rows > 64) {
    FusedSample fs{tokens, lse, logq, extra, 0.f, 0};
    return draft_step_impl(v, w, anchor, logits, workspace, draft, nullptr, 0, st, &fs);
  }
  // otherwise the sampler needs the logits (the same tokens as ldr_sample)
  if (!logits) return LDR_EINVAL;
  // T > 0 on the tiled head: the chunk log-masses in its epilogue, then the
  // sampler's chunk draw
  if (w->lm_head_tiled && rows > 64) {
    FusedSample fs{tokens, lse, logq, extra, temperature, sample_plan(rows, s.vocab).ldL};
    const int rc = draft_step_impl(v, w, anchor, logits, workspace, draft, nullptr, 0, st, &fs);
    if (rc != LDR_OK) return rc;
    return launch_sample_finish(logits, rows, s.vocab, temperature, seed, step, extra, tokens,
                                lse, logq, st) == hipSuccess
               ? LDR_OK : LDR_EHIP;
  }
  const int rc = draft_step_impl(v, w, anchor, logits, workspace, draft, nullptr, 0, st);
  if (rc != LDR_OK) return rc;
  return launch_sample(logits, rows, s.vocab, temperature, 0, seed, step, tokens, lse, logq,
                       extra, align_up(sample_part_bytes(rows, s.vocab)), st) == hipSuccess
             ? LDR_OK : LDR_EHIP;
}

int ldr_draft_step_events(const ldr_views* v, const ldr_weights* w, const int32_t* anchor,
                          float* logits, void* workspace, size_t workspace_bytes,
                          void* const* events, int32_t n_events, void* stream) {
  if (!events) return LDR_EINVAL;
  return draft_step_impl(v, w, anchor, logits, workspace, workspace_bytes, events, n_events,
                         static_cast<hipStream_t>(stream));
}

size_t ldr_sample_workspace_bytes(int32_t rows, int32_t vocab) {
  if (rows <= 0 || vocab <= 0) return 0;
  return align_up(sample_part_bytes(rows, vocab)) + align_up((size_t)rows * 8);
}

int ldr_sample(const float* logits, int32_t rows, int32_t vocab, float temperature,
               int32_t top_k, uint64_t seed, uint64_t step, int32_t* tokens, float* lse,
               float* logq, void* workspace, size_t workspace_bytes, void* stream) {
  if (!logits || !tokens || !lse || !logq || !workspace) return LDR_EINVAL;
  if (rows <= 0 || vocab <= 0 || !(temperature >= 0.f) || std::isinf(temperature))
    return LDR_EINVAL;
  if (top_k < 0) return LDR_EINVAL;
  if (workspace_bytes < ldr_sample_workspace_bytes(rows, vocab) || !aligned(workspace, 16))
    return LDR_EINVAL;
  return launch_sample(logits, rows, vocab, temperature, top_k, seed, step, tokens, lse, logq,
                       workspace, align_up(sample_part_bytes(rows, vocab)),
                       static_cast<hipStream_t>(stream)) == hipSuccess
             ? LDR_OK : LDR_EHIP;
}

int ldr_sample_noalloc(const float* logits, int32_t rows, int32_t vocab, float temperature,
                       int32_t top_k, uint64_t seed, uint64_t step, int32_t* tokens, float* lse,
                       float* logq, void* stream) {
  if (!logits || !tokens || !lse || !logq) return LDR_EINVAL;
  if (rows <= 0 || vocab <= 0 || !(temperature >= 0.f) || std::isinf(temperature))
    return LDR_EINVAL;
  if (top_k < 0) return LDR_EINVAL;
  if (ldr_sample_workspace_bytes(rows, vocab) > LDR_NOALLOC_SCRATCH_BYTES) return LDR_ESCRATCH;
  void* ws = nullptr;
  if (noalloc_scratch(&ws) != hipSuccess) return LDR_EHIP;
  return launch_sample(logits, rows, vocab, temperature, top_k, seed, step, tokens, lse, logq, ws,
                       align_up(sample_part_bytes(rows, vocab)),
                       static_cast<hipStream_t>(stream)) == hipSuccess
             ? LDR_OK : LDR_EHIP;
}

int ldr_sample_markov(float* logits, int32_t batch, int32_t block, int32_t vocab,
                      const int32_t* anchor, const void* E_c, const void* W_c, int32_t rank,
                      int32_t dtype, float temperature, int32_t top_k, uint64_t seed,
                      uint64_t step, int32_t* tokens, float* lse, float* logq, void* workspace,
                      size_t workspace_bytes, void* stream) {
  if (!logits || !anchor || !E_c || !W_c || !tokens || !lse || !logq || !workspace)
    return LDR_EINVAL;
  if (batch <= 0 || block <= 0 || vocab <= 0 || !(temperature >= 0.f) || std::isinf(temperature))
    return LDR_EINVAL;
  if (top_k < 0 || (dtype != LDR_BF16 && dtype != LDR_F32)) return LDR_EINVAL;
  if (rank <= 0 || rank > 256 || rank % 8) return LDR_EINVAL;
  if (!aligned(E_c, 16) || !aligned(W_c, 16) || !aligned(workspace, 16)) return LDR_EINVAL;
  if (workspace_bytes < ldr_sample_workspace_bytes(batch, vocab)) return LDR_EINVAL;
  return launch_sample_markov(logits, batch, block, vocab, anchor, E_c, W_c, rank, dtype,
                              temperature, top_k, seed, step, tokens, lse, logq, workspace,
                              align_up(sample_part_bytes(batch, vocab)),
                              static_cast<hipStream_t>(stream)) == hipSuccess
             ? LDR_OK : LDR_EHIP;
}

size_t ldr_verify_workspace_bytes(int32_t batch, int32_t block, int32_t vocab) {
  if (batch <= 0 || block <= 0 || vocab <= 0) return 0;
  return verify_workspace_bytes(batch, block, vocab);
}

int ldr_verify(const float* target_logits, const float* draft_logits, const float* draft_lse,
               const int32_t* draft_tokens, int32_t batch, int32_t block, int32_t vocab,
               float temperature, int32_t top_k, uint64_t seed, uint64_t step,
               int32_t* accepted, int32_t* next_token, int32_t* n_new, void* workspace,
               size_t workspace_bytes, void* stream) {
  if (!target_logits || !draft_tokens || !accepted || !next_token || !n_new || !workspace)
    return LDR_EINVAL;
  if (batch <= 0 || block <= 0 || vocab <= 0 || !(temperature >= 0.f) || std::isinf(temperature))
    return LDR_EINVAL;
  if (temperature > 0.f && (!draft_logits || !draft_lse)) return LDR_EINVAL;
  if (top_k < 0) return LDR_EINVAL;
  if (workspace_bytes < ldr_verify_workspace_bytes(batch, block, vocab) || !aligned(workspace, 16))
    return LDR_EINVAL;
  return launch_verify(target_logits, draft_logits, draft_tokens, draft_lse, batch, block, vocab,
                       temperature, top_k, seed, step, accepted, next_token, n_new, workspace,
                       static_cast<hipStream_t>(stream)) == hipSuccess
             ? LDR_OK : LDR_EHIP;
}

int ldr_gumbel_fill(uint64_t seed, uint64_t step, int32_t noise_stream, int32_t rows,
                    int32_t vocab, float* out, void* stream) {
  if (!out || rows <= 0 || vocab <= 0 || noise_stream < 0 || noise_stream > 3) return LDR_EINVAL;
  return launch_gumbel_fill(seed, step, noise_stream, rows, vocab, out,
                            static_cast<hipStream_t>(stream)) == hipSuccess ? LDR_OK : LDR_EHIP;
}

}  // extern "C"
