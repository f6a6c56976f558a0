/*
 * ldr.h -- fixed-cost speculative drafting on one MI355X (gfx950).
 *
 * C ABI of the drafting step of "Efficient speculative decoding with a
 * fixed-cost parallel drafter" (LongSpark): the fixed-size context views of
 * Sec. 2.2 and their incremental maintenance (App. A.2, Eq. 10-11), the
 * block-diffusion drafter forward (Sec. 2.3, Eq. 4 and Eq. 6, App. A.1,
 * App. B.1) and per-position sampling of the factorised proposal (Eq. 8);
 * around it, the ablation variants' views (Sec. 3.4), the low-rank Markov
 * correction of the proposal (Eq. 7) and the speculative verification that
 * closes a round (Eq. 1-2).
 *
 * Conventions shared by every entry point:
 *  - Pointers marked "dev" are device memory owned by the caller (for
 *    example PyTorch tensors). The library never frees them and never keeps
 *    them beyond the call, except the arena, position and G pointers that
 *    ldr_views_init records in the handle.
 *  - `stream` is a hipStream_t (NULL: the legacy default stream). Every call
 *    that takes one only enqueues work on it and returns without waiting.
 *  - Host-side validation is synchronous: on a bad argument nothing is
 *    enqueued and LDR_EINVAL is returned. A failed kernel launch returns
 *    LDR_EHIP. Errors detected on the device (an out-of-range row count) set
 *    a sticky flag read by ldr_views_status.
 *  - Matrices are row-major in the nn.Linear [out][in] layout. "dtype" is the
 *    configuration's element type (fp32 or bf16) of weights, window rows,
 *    summary queries and boundary states; summary values and
 *    log-normalizers, logits and sampler outputs are always fp32.
 *  - All 16-byte-vector accesses need 16-byte-aligned pointers and row
 *    lengths; the library checks this and returns LDR_EINVAL otherwise.
 */
#ifndef LDR_H
#define LDR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum ldr_status {
  LDR_OK = 0,
  LDR_EINVAL = -1,  /* bad argument, shape or alignment (host check)        */
  LDR_ERANGE = -2,  /* a per-sequence row count outside [0, max_new]        */
  LDR_EHIP = -3,    /* a HIP runtime call or kernel launch failed           */
  LDR_ENOMEM = -4,  /* the small host/device bookkeeping allocation failed  */
  LDR_ESCRATCH = -5 /* the call needs more than the static scratch holds    */
};

enum ldr_dtype { LDR_F32 = 0, LDR_BF16 = 1 };

/* Views an ablation variant leaves out (Sec. 3.4, App. D.3): bits of
 * ldr_config.drop_views. A dropped view is neither kept nor read: its arena
 * region has zero bytes, the update skips it and the draft step attends to
 * the other sources only (no window rows; no summary entries), or takes
 * c_t = 0 without the boundary-fusion GEMM. */
enum ldr_view_drop {
  LDR_DROP_WINDOW = 1,    /* no recent K/V window                          */
  LDR_DROP_SUMMARY = 2,   /* no global summary (G may then be NULL)        */
  LDR_DROP_BOUNDARY = 4   /* no boundary state (h may then be NULL)        */
};

/* Drafter shape (App. B.1: D = 5 Qwen3-style layers, W = 256, R = 16). */
typedef struct ldr_config {
  int32_t hidden;        /* model width                                        */
  int32_t n_q_heads;     /* Hq                                                 */
  int32_t n_kv_heads;    /* Hkv, divides Hq; q head h reads kv group h/(Hq/Hkv) */
  int32_t head_dim;      /* d, 64 or 128                                       */
  int32_t mlp;           /* SwiGLU intermediate width                          */
  int32_t vocab;         /* V                                                  */
  int32_t n_layers;      /* D: draft layers, each paired with one window and
                            one summary bank (Sec. 2.3)                        */
  int32_t n_feat_layers; /* L_b: boundary hidden states fused into c_t         */
  int32_t block;         /* B: slots = proposals per round, 1..16              */
  int32_t window;        /* W: recent K/V rows kept per layer                  */
  int32_t summary;       /* R: summary queries per layer and query head        */
  int32_t dtype;         /* enum ldr_dtype                                     */
  float rope_theta;      /* rotary base                                        */
  float ntk_alpha;       /* fixed NTK scaling: base = theta * alpha^(d/(d-2))  */
  float rms_eps;         /* RMSNorm epsilon                                    */
  int32_t drop_views;    /* 0 (the full drafter) or a sum of ldr_view_drop bits
                            that keeps at least one view                     */
  int32_t pool_slots;    /* 0: the learned-query summary (Eq. 5). P > 0: the
                            mean-pooled summary instead (the views as the
                            configurations word them): two banks of P ring
                            slots, slot c mod P holding the mean K and V row
                            of chunk c (pool_stride rows); P % 32 == 0; the
                            summary queries G and `summary` are then unused */
  int32_t pool_stride[2];/* rows per chunk of the two banks, each >= 1      */
} ldr_config;

/* Device pointers of one draft layer (Qwen3-style block, App. B.1). */
typedef struct ldr_layer_weights {
  const void* in_norm;   /* dev [hidden]                 pre-attention RMSNorm gain */
  const void* wqkv;      /* dev [(Hq+2Hkv)d][hidden]     rows: q heads, k heads, v heads */
  const void* q_norm;    /* dev [d]                      per-head q RMSNorm gain  */
  const void* k_norm;    /* dev [d]                      per-head k RMSNorm gain  */
  const void* wo;        /* dev [hidden][Hq d]                                     */
  const void* post_norm; /* dev [hidden]                 pre-MLP RMSNorm gain     */
  const void* w_gate_up; /* dev [2 mlp][hidden]          rows: gate, then up      */
  const void* w_down;    /* dev [hidden][mlp]                                      */
} ldr_layer_weights;

/* Device pointers of the drafter (all in the configuration dtype). The
 * embedding, final norm and vocabulary head are the target's, frozen
 * (Sec. 2.3); embed and lm_head may be the same pointer. */
typedef struct ldr_weights {
  const void* embed;       /* dev [V][hidden]                                   */
  const void* mask_emb;    /* dev [hidden]      the mask-token embedding         */
  const void* pos_emb;     /* dev [B][hidden]   within-block positional encoding */
  const void* fc_w;        /* dev [hidden][L_b hidden]  boundary fusion          */
  const void* fc_norm;     /* dev [hidden]      boundary fusion RMSNorm gain     */
  const void* final_norm;  /* dev [hidden]                                       */
  const void* lm_head;     /* dev [V][hidden]                                    */
  const ldr_layer_weights* layers; /* host array of n_layers entries            */
  const void* lm_head_tiled; /* dev, optional: lm_head in the tiled layout of
                                ldr_tile_matrix (ldr_tiled_bytes(V, hidden)
                                bytes), bf16 configurations with hidden % 128
                                == 0 only; read when batch * B > 64 (smaller
                                steps use lm_head); NULL: the head always reads
                                lm_head. Same logits up to fp32 summation
                                order. */
} ldr_weights;

typedef struct ldr_views ldr_views; /* opaque host handle */

/* Per-sequence bytes of the fixed-size views (Sec. 2.4, Fixed-cost
 * complexity): window K [D][Hkv][W][d] and window V stored transposed,
 * [D][Hkv][d][W] (dtype; slot p mod W of position p; with the mean-pooled
 * summary each (layer, group) holds W + 2P rows: the window, then bank 0's
 * and bank 1's slot means, and fp32 sums of the open chunks [D][Hkv][2][2][d]
 * follow the boundary region), summary values
 * [D][Hq][R][d] and log-normalizers [D][Hq][R] (fp32), boundary states
 * [L_b][hidden] (dtype), each region 256-byte aligned; a view the
 * configuration drops has zero bytes. No term depends on the prefix length.
 * Returns 0 for an invalid configuration. */
size_t ldr_views_state_bytes(const ldr_config* cfg);

/* Byte stride between sequences in the arena (state bytes rounded up to 256),
 * so an arena for `batch` sequences needs batch * stride bytes. */
size_t ldr_views_stride_bytes(const ldr_config* cfg);

/* Byte offsets, inside one sequence's slot, of the window K, window V,
 * summary values, summary log-normalizers and boundary states (5 entries
 * written to `offsets`). Returns LDR_OK or LDR_EINVAL. */
int ldr_views_layout(const ldr_config* cfg, size_t offsets[5]);

/* Bytes of a bf16 [rows][cols] matrix in the tiled layout below. */
size_t ldr_tiled_bytes(int32_t rows, int32_t cols);

/* Enqueues a tiled copy of the row-major bf16 matrix src [rows][cols] (dev,
 * row stride ld elements) into dst (dev, dst_bytes >= ldr_tiled_bytes): column
 * blocks of 32, element (r, c) at element offset (c / 32) * R * 32 + r * 32 +
 * c % 32 with R = rows rounded up to a multiple of 256; rows from `rows` to R
 * are zero. One K block of any run of weight rows is then one contiguous
 * stretch for the vocabulary head's GEMM (App. B.1 shares the target's head,
 * V x hidden, so this is a one-time copy of a frozen weight). Needs
 * cols % 32 == 0, ld >= cols and 16-byte aligned pointers and rows (ld % 8
 * == 0), else LDR_EINVAL. The caller owns both buffers. */
int ldr_tile_matrix(const void* src, int32_t rows, int32_t cols, int64_t ld, void* dst,
                    size_t dst_bytes, void* stream);

/* Workspace bytes ldr_draft_step needs for `batch` sequences. */
size_t ldr_workspace_bytes(const ldr_config* cfg, int32_t batch);

/* Validates a configuration: LDR_OK or LDR_EINVAL. */
int ldr_config_check(const ldr_config* cfg);

/* Creates a views handle for `batch` sequences over a caller-owned arena and
 * enqueues its reset to the empty state (Sec. 2.2; App. A.2): every position
 * counter 0, summary log-normalizers -inf, summary values, window and
 * boundary states 0. Then, if max_prefix > 0, ingests a first prefix chunk
 * exactly as ldr_views_update would (the summary is initialised over the
 * prefix once, at prefill: Sec. 2.2, Fig. "global-summary").
 *   arena      dev [batch][stride] bytes, 256-byte aligned (kept in the handle)
 *   pos        dev int64 [batch]: rows ingested per sequence, t (kept)
 *   G          dev [D][Hq][R][d] dtype: the fixed summary queries (kept); may be
 *              NULL when the configuration has no learned summary
 *              (LDR_DROP_SUMMARY, or pool_slots > 0)
 *   n_prefix   dev int32 [batch] rows per sequence in the chunk, or NULL
 *   K_prefix, V_prefix  dev [batch][max_prefix][D][Hkv][d] dtype
 *   h_boundary dev [batch][L_b][hidden] dtype: boundary states after it (may be
 *              NULL with LDR_DROP_BOUNDARY)
 * The handle also owns a 256-byte device status block (the sticky flags and
 * the update's commit counter), freed by ldr_views_destroy. */
int ldr_views_init(ldr_views** out, const ldr_config* cfg, int32_t batch, void* arena,
                   int64_t* pos, const void* G, const int32_t* n_prefix, int32_t max_prefix,
                   const void* K_prefix, const void* V_prefix, const void* h_boundary,
                   void* stream);

/* Ingests the target K/V rows committed by one verification pass (Sec. 2.4,
 * Inference; App. A.2). For every sequence b with n = n_new[b] rows:
 *  - row r (position t_b + r) is written to window slot (t_b + r) mod W for
 *    every layer (only the last min(n, W) rows can survive, and only they
 *    are written);
 *  - the rows form the set N of Eq. 10 for every (layer j, query head h,
 *    summary query r): s = G[j,h,r] . k / sqrt(d) over the head's K/V group,
 *    eta_N and m_N by log-sum-exp with max subtraction, merged into (eta, m)
 *    by Eq. 11;
 *  - with the mean-pooled summary (pool_slots = P > 0) instead of the
 *    previous point: for each bank of stride S, the slot c mod P of every
 *    chunk c the rows reach takes the mean of chunk c's rows so far (fp32
 *    sums, the open chunk continuing from its stored sums), K and V;
 *  - the boundary states become h_new[b];
 *  - t_b += n.
 * A view the configuration drops (drop_views) is left out of this list.
 * n = 0 leaves that sequence's views and t bit-identical (App. A.2). A count
 * outside [0, max_new] leaves the sequence unchanged and sets the sticky
 * LDR_ERANGE flag. Calls on one handle must be ordered (one stream, or
 * streams joined by events): t is advanced by the last workgroup of the
 * update, counted in the handle's status block.
 *   n_new       dev int32 [batch]
 *   K_new, V_new dev [batch][max_new][D][Hkv][d] dtype (row r of sequence b at
 *               [b][r]; rows r >= n_new[b] are ignored)
 *   h_new       dev [batch][L_b][hidden] dtype (may be NULL with LDR_DROP_BOUNDARY) */
int ldr_views_update(ldr_views* v, const int32_t* n_new, int32_t max_new, const void* K_new,
                     const void* V_new, const void* h_new, void* stream);

/* Waits for `stream` and returns the sticky device status: LDR_OK,
 * LDR_ERANGE once any update saw an out-of-range row count, else LDR_EINVAL
 * once any draft step saw an anchor outside [0, V) (that slot then used token
 * 0). Clears the status if `clear` is nonzero. */
int ldr_views_status(ldr_views* v, int clear, void* stream);

/* Frees the handle and its status word; the arena, pos and G stay the
 * caller's. NULL is ignored. */
void ldr_views_destroy(ldr_views* v);

/* One block proposal (Eq. 4; Sec. 2.3; App. A.1): base logits z^(0) of the B
 * slots of every sequence, from the views alone.
 *  c_b = RMSNorm(W_fc [h_0; ...; h_{L_b-1}]), x_{b,i} = E[u_i] + P_i + c_b with
 *  u_0 = anchor[b] and u_i = the mask embedding for i >= 1; slot i sits at
 *  absolute position t_b + i. Then D pre-norm layers: per-head q/k RMSNorm and
 *  rotary embedding on the block's q and k, attention of every query head h
 *  over [block k; window K of layer j; G[j,h]] with values
 *  [block v; window V; M[j,h]] under ONE softmax (Eq. 6), no mask among the
 *  slots, window slots masked while t_b < W, summary entries masked while
 *  t_b = 0; SwiGLU MLP. Final RMSNorm and vocabulary head.
 *   anchor    dev int32 [batch], each in [0, V); an anchor outside it is
 *             replaced by token 0 and recorded in the views status
 *   logits    dev fp32 [batch][B][V] (row b*B + i proposes y_{i+1})
 *   workspace dev, at least ldr_workspace_bytes(cfg, batch) bytes, 256-aligned;
 *             its contents are scratch, owned by the caller. */
int ldr_draft_step(const ldr_views* v, const ldr_weights* w, const int32_t* anchor,
                   float* logits, void* workspace, size_t workspace_bytes, void* stream);

/* Kernel launches of one draft step, in order. */
enum ldr_launch_kind {
  LDR_LAUNCH_FC_GEMM = 0,      /* boundary fusion W_fc (split-K partials)          */
  LDR_LAUNCH_SLOT_INIT = 1,    /* c_t norm, slot inputs, first pre-norm, RoPE table */
  LDR_LAUNCH_QKV_GEMM = 2,     /* per layer: QKV projection                         */
  LDR_LAUNCH_ATTENTION = 3,    /* per layer: block-view attention (Eq. 6); bf16: it
                                  also finishes q, k, v from the QKV partials       */
  LDR_LAUNCH_O_GEMM = 4,       /* per layer: output projection                      */
  LDR_LAUNCH_POST_NORM = 5,    /* per layer: residual add + pre-MLP RMSNorm         */
  LDR_LAUNCH_GATE_UP_GEMM = 6, /* per layer: gate/up projection + SwiGLU            */
  LDR_LAUNCH_DOWN_GEMM = 7,    /* per layer: down projection                        */
  LDR_LAUNCH_NEXT_NORM = 8,    /* per layer: residual add + next (or final) RMSNorm */
  LDR_LAUNCH_LM_HEAD = 9,      /* vocabulary head, fp32 logits                      */
  LDR_LAUNCH_QKV_FINISH = 10   /* per layer (fp32 models): QKV split-K sum, q/k
                                  RMSNorm, RoPE                                     */
};

/* Number of kernel launches of ldr_draft_step for this configuration
 * (LDR_EINVAL if invalid); writes the kind of each, in order, to
 * kinds[0 .. max_kinds). kinds may be NULL. */
int32_t ldr_draft_step_launches(const ldr_config* cfg, int32_t* kinds, int32_t max_kinds);

/* ldr_draft_step that also records caller-created hipEvent_t events on
 * `stream`: events[i] right before launch i and events[n] after the last
 * launch, n = ldr_draft_step_launches(cfg). n_events must be n + 1; NULL
 * entries are skipped. For timing single kernels of the step. */
int ldr_draft_step_events(const ldr_views* v, const ldr_weights* w, const int32_t* anchor,
                          float* logits, void* workspace, size_t workspace_bytes,
                          void* const* events, int32_t n_events, void* stream);

/* Workspace bytes ldr_draft_step_sample needs for `batch` sequences. */
size_t ldr_draft_step_sample_workspace_bytes(const ldr_config* cfg, int32_t batch);

/* ldr_draft_step followed by per-position sampling of every row (Eq. 4 and
 * Eq. 8): tokens, lse and logq are those of ldr_sample(logits, batch * B, V,
 * temperature, top_k = 0, seed, step) on the step's logits, bit for bit. Greedy
 * steps (temperature 0) whose head reads its tiled copy (w->lm_head_tiled set
 * and batch * B > 64) take the argmax in the head's epilogue, from the fp32
 * logits it has just computed, so the logits need not be written
 * (logits = NULL). Sampled steps on the tiled head form the two-level draw's
 * 16-token chunk log-masses in the head's epilogue, with the bits ldr_sample's
 * pass over the written logits gives them, then run ldr_sample's chunk draw;
 * other steps run the head and then ldr_sample's kernels. Both need the
 * logits.
 *   logits  dev fp32 [batch][B][V], or NULL on the fused greedy path
 *   tokens  dev int32 [batch][B]; lse, logq dev fp32 [batch][B]
 *   workspace dev, ldr_draft_step_sample_workspace_bytes(cfg, batch) bytes,
 *           256-byte aligned.
 * LDR_EINVAL on a bad argument (as ldr_draft_step and ldr_sample), or NULL
 * logits off the fused greedy path. */
int ldr_draft_step_sample(const ldr_views* v, const ldr_weights* w, const int32_t* anchor,
                          float* logits, float temperature, uint64_t seed, uint64_t step,
                          int32_t* tokens, float* lse, float* logq, void* workspace,
                          size_t workspace_bytes, void* stream);

/* Workspace bytes ldr_sample needs for `rows` rows of `vocab` logits. */
size_t ldr_sample_workspace_bytes(int32_t rows, int32_t vocab);

/* Per-position sampling of the factorised proposal (Eq. 8), one row at a
 * time and independently. temperature = 0: tokens[r] = argmax z (lowest index
 * on ties), lse[r] = that maximum, logq[r] = 0. temperature T > 0: support S =
 * all V tokens (top_k = 0) or the top_k largest logits (lower index first on
 * ties), and a two-level Gumbel-max, an exact draw from softmax(z/T) over S:
 * the vocabulary is cut into chunks of 16 tokens (chunk c = tokens 16c ..
 * 16c + 15), chunk c has log-mass L_c = log sum_{v in c, v in S} exp(z_v / T)
 * (fp32), the chunk is the first argmax of fl(L_c + h_c) and the token the
 * first argmax over that chunk's support tokens of fl(fl(z_v / T) + g_v).
 * Noise: Philox4x32-10 with key (seed mod 2^32, seed div 2^32) and counter
 * (e div 4, r, step mod 2^32, (step div 2^32) mod 2^30 + 2^30 s), word e mod 4,
 * u = (2 (bits >> 9) + 1) 2^-24 and -log(-log(u)) with a fixed-operation fp32
 * logarithm: g_v is entry v of stream s = 0, h_c entry c of stream s = 3 (a
 * step is unique below 2^62). The token keys are reproducible bit for bit on
 * any IEEE machine; L_c is an fp32 sum whose last bits depend on the order of
 * its 16 terms (fixed here). lse[r] = log sum_{v in S} exp(z_v / T);
 * logq[r] = z_y / T - lse[r].
 * top_k >= vocab is the full vocabulary; a negative top_k is LDR_EINVAL. With
 * 0 < top_k < vocab an extra pass per row selects the exact top_k support
 * (-0 and +0 compare equal).
 *   logits dev fp32 [rows][vocab]; tokens dev int32 [rows]; lse, logq dev fp32 [rows]
 *   workspace dev, ldr_sample_workspace_bytes(rows, vocab) bytes. */
int ldr_sample(const float* logits, int32_t rows, int32_t vocab, float temperature,
               int32_t top_k, uint64_t seed, uint64_t step, int32_t* tokens, float* lse,
               float* logq, void* workspace, size_t workspace_bytes, void* stream);

/* Bytes of the library's static device scratch behind ldr_sample_noalloc. */
#define LDR_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)

/* ldr_sample for callers that cannot allocate device memory (code under HIP
 * graph capture, serving loops that forbid allocation): the same kernels,
 * tokens, lse and logq as ldr_sample with the same arguments, bit for bit, with
 * the chunk log-masses, the partials and the top-k supports in a file-scope
 * device array of LDR_NOALLOC_SCRATCH_BYTES bytes instead of a caller
 * workspace. Each GPU the library runs on holds its own copy of that array
 * until the process ends; its address is looked up once per device, on the
 * first call with that device current. The call allocates nothing (no
 * hipMalloc, no library routine that allocates). Every call on one GPU shares
 * that GPU's array and leaves its contents behind; nothing in it needs to
 * start at zero (each launch writes every entry it later reads), but calls
 * whose stream work overlaps on the same GPU race on it: serialise them (one
 * stream, or events). Requests with ldr_sample_workspace_bytes(rows, vocab) >
 * LDR_NOALLOC_SCRATCH_BYTES (about 430 rows of a 151936-token vocabulary)
 * return LDR_ESCRATCH before anything is enqueued; bad arguments return
 * LDR_EINVAL as in ldr_sample.
 *   logits dev fp32 [rows][vocab]; tokens dev int32 [rows]; lse, logq dev fp32 [rows] */
int ldr_sample_noalloc(const float* logits, int32_t rows, int32_t vocab, float temperature,
                       int32_t top_k, uint64_t seed, uint64_t step, int32_t* tokens, float* lse,
                       float* logq, void* stream);

/* Markov-corrected sampling (Eq. 7-8; the low-rank sequential correction the
 * paper takes from DSpark). For every sequence b and position i = 1 .. B in
 * order, with y_0 = anchor[b]:
 *   z_i <- fl(z_i + c),  c[v] = sum_{k = 0 .. rank-1, in order} fl(W_c[v][k] E_c[y_{i-1}][k])
 * with every product and partial sum an fp32 operation (none fused), then
 * y_i, lse and log q of row b * block + i - 1 exactly as ldr_sample computes
 * them for that row of the corrected logits (same noise counter, temperature
 * and top_k rules). The positions are sampled one after the other (each
 * correction needs the previous token); the sequences in parallel.
 *   logits   dev fp32 [batch][block][vocab]: the base logits z^(0) on entry,
 *            the corrected logits z when the stream reaches the end of the call
 *   anchor   dev int32 [batch] (outside [0, vocab) reads embedding row 0)
 *   E_c, W_c dev [vocab][rank] in `dtype` (enum ldr_dtype): correction
 *            embedding and output mapping; rank > 0, a multiple of 8, at
 *            most 256
 *   tokens   dev int32 [batch][block]; lse, logq dev fp32 [batch][block]
 *   workspace dev, ldr_sample_workspace_bytes(batch, vocab) bytes.
 * LDR_EINVAL on a bad argument (as ldr_sample, plus the rank and dtype). */
int ldr_sample_markov(float* logits, int32_t batch, int32_t block, int32_t vocab,
                      const int32_t* anchor, const void* E_c, const void* W_c, int32_t rank,
                      int32_t dtype, float temperature, int32_t top_k, uint64_t seed,
                      uint64_t step, int32_t* tokens, float* lse, float* logq, void* workspace,
                      size_t workspace_bytes, void* stream);

/* Workspace bytes ldr_verify needs (0 on a non-positive size). */
size_t ldr_verify_workspace_bytes(int32_t batch, int32_t block, int32_t vocab);

/* Speculative verification of one drafted block per sequence (Eq. 1-2), the
 * step that closes a round. The target has scored [a, y_1 .. y_B] in one pass:
 * target row j of sequence b is p_{j+1} = softmax(P[b][j] / T), j = 0 .. B; the
 * proposal q_i is softmax(z[b][i-1] / T) over the drafting sampler's support
 * (the whole vocabulary when top_k is 0 or >= vocab, else the top_k largest
 * logits, lower index first on ties) and 0 outside it: the logits and top_k
 * ldr_sample or ldr_sample_markov drew y from, with the lse it wrote.
 * Candidates are tested in order: y_i is accepted when u_i < p_i(y_i) / q_i(y_i);
 * a candidate outside [0, vocab) or outside the support is rejected. At the
 * first rejection, i, the round emits the first argmax of log w_v + g_v over
 * the residual w_v = [p_i(v) - q_i(v)]_+, every token with w_v > 0 as computed
 * in fp32; after B acceptances, and when w has no positive entry, it emits the
 * first argmax of fl(fl(P_v / T) + g_v) over the row (a one-level Gumbel-max).
 * Noise: ldr_sample's Philox4x32-10 layout with the top two bits of the
 * last counter word set to a stream: u_i is word 0 of counter (i - 1, b, ...)
 * in stream 1, g_v token v of row b in stream 2; both through
 * u = (2 (bits >> 9) + 1) 2^-24, and g = -log(-log(u)) with ldr_sample's
 * fixed-operation logarithm. T = 0 verifies greedily: y_i is accepted when it
 * is the first argmax of P[b][i-1], and the round emits the first argmax of
 * the row where it stops (draft_logits, draft_lse and top_k are not read and
 * draft_logits / draft_lse may be NULL). The ratio, the residual and the
 * target's log-normalisers are fp32, so decisions closer than their rounding
 * (a ratio within ~1e-6 of u, residual entries within ~1e-6 of p) may differ
 * from the exact ones.
 *   target_logits dev fp32 [batch][block + 1][vocab]
 *   draft_logits  dev fp32 [batch][block][vocab]; draft_lse dev fp32 [batch][block]
 *   draft_tokens  dev int32 [batch][block]
 *   top_k         the sampler's support size (0: the whole vocabulary)
 *   accepted      dev int32 [batch]: r, the accepted candidates (0 .. block)
 *   next_token    dev int32 [batch]: the emitted token (the next anchor)
 *   n_new         dev int32 [batch]: r + 1, the rows the prefix advances by (the
 *                 per-sequence row count of the next ldr_views_update)
 *   workspace     dev, ldr_verify_workspace_bytes(batch, block, vocab) bytes.
 * LDR_EINVAL on a NULL pointer, a non-positive size, a negative top_k, a
 * negative, NaN or infinite temperature, or a short or misaligned workspace. */
int ldr_verify(const float* target_logits, const float* draft_logits, const float* draft_lse,
               const int32_t* draft_tokens, int32_t batch, int32_t block, int32_t vocab,
               float temperature, int32_t top_k, uint64_t seed, uint64_t step,
               int32_t* accepted, int32_t* next_token, int32_t* n_new, void* workspace,
               size_t workspace_bytes, void* stream);

/* Writes Gumbel noise of the samplers' layout: out[r][e] = -log(-log(u)) of
 * entry e of row r in noise stream noise_stream (0: ldr_sample's token noise
 * g, 3: its chunk noise h, 1 and 2: ldr_verify's), for rows [0, rows) and
 * entries [0, vocab). out dev fp32 [rows][vocab]. LDR_EINVAL on a NULL out, a
 * non-positive size or a stream outside 0 .. 3. */
int ldr_gumbel_fill(uint64_t seed, uint64_t step, int32_t noise_stream, int32_t rows,
                    int32_t vocab, float* out, void* stream);

/* A static string naming a status code. */
const char* ldr_strerror(int status);

#ifdef __cplusplus
}
#endif
#endif /* LDR_H */
