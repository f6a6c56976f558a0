"""Oracle for the block-diffusion drafter forward (Eq. 4, Eq. 6; Sec. 2.3;
App. A.1; App. B.1), float64.

One call proposes the base logits z^(0)_{1:B} of one sequence from its views
alone:

1. boundary fusion: c = RMSNorm(W_fc [h_0; ...; h_{L_b-1}]) with gain g_fc;
2. slot init: x_i = E[u_i] + P_i + c, u_0 = the committed token a, u_i (i >= 1)
   = the mask embedding; slot i sits at absolute position t + i;
3. D Qwen3-style layers; layer j attends, for every query head h, over one
   concatenation [block keys; window keys of layer j; G[j,h]] with values
   [block values; window values; M[j,h]] and ONE softmax across the three
   sources, no mask among the block slots (Eq. 6, App. A.1);
4. frozen final RMSNorm and vocabulary head -> fp64 logits [B][V].

Readings where the paper is silent (Qwen3 conventions): pre-norm RMSNorm
with eps from the shape, per-head q/k RMSNorm on the drafter's own q and
block k, rotate-half RoPE on q and block k at absolute positions with base
theta * alpha^(d/(d-2)); window keys are used as stored (already rotated
target-cache rows) and G is never rotated; SwiGLU MLP.
"""
from __future__ import annotations

import numpy as np
import scipy.special

from . import views as _views


def rmsnorm(x, g, eps):
    """x / sqrt(mean(x^2) + eps) * g over the last axis."""
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * g


def silu(x):
    return x / (1.0 + np.exp(-x))


def rope_base(s) -> float:
    """Rotary base with fixed NTK scaling by alpha (alpha = 1: plain theta)."""
    d = s.head_dim
    return s.rope_theta * s.ntk_alpha ** (d / (d - 2))


def rope(x, pos, base):
    """Rotate-half rotary embedding. x [n][H][d], pos [n] absolute positions.
    Pair (e, e + d/2) is rotated by angle pos * base^(-2e/d)."""
    d = x.shape[-1]
    half = d // 2
    inv = base ** (-(np.arange(half) * 2.0) / d)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv[None, :]   # [n][half]
    cos, sin = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * cos - x2 * sin, x1 * sin + x2 * cos], axis=-1)


def block_attention(q, kb, vb, Kw, Vw, valid, G, M, has_summary, pooled=()):
    """Eq. 6 for one query head: q [B][d] against keys [kb; Kw[valid]; G]
    and values [vb; Vw[valid]; M] with one softmax, scale 1/sqrt(d).
    `pooled`: (keys, values) of the mean-pooled summary's valid slots, which
    join the concatenation in place of G and M."""
    d = q.shape[-1]
    keys = [kb, Kw[valid]]
    vals = [vb, Vw[valid]]
    if has_summary:
        keys.append(G)
        vals.append(M)
    for pk, pv in pooled:
        keys.append(pk)
        vals.append(pv)
    K = np.concatenate(keys, axis=0)
    V = np.concatenate(vals, axis=0)
    p = scipy.special.softmax(q @ K.T / np.sqrt(d), axis=-1)
    return p @ V


def boundary_fusion(s, Wt, h):
    """c_t = RMSNorm(W_fc [h_0; ...; h_{L_b-1}]) (Sec. 2.2, boundary state)."""
    return rmsnorm(Wt["fc_w"] @ h.reshape(-1), Wt["fc_norm"], s.rms_eps)


def slot_init(s, Wt, c, anchor):
    """x_i = E[u_i] + P_i + c with u_0 = a and u_i = mask for i >= 1 (Sec. 2.3)."""
    x = np.empty((s.block, s.hidden))
    x[0] = Wt["embed"][anchor]
    x[1:] = Wt["mask_emb"]
    return x + Wt["pos_emb"] + c


def layer(s, L, x, st: _views.ViewState, G, j):
    """One Qwen3-style draft layer j over the B slots (pre-norm, residual)."""
    B, Hq, Hkv, d = s.block, s.n_q_heads, s.n_kv_heads, s.head_dim
    rep = Hq // Hkv
    n = rmsnorm(x, L["in_norm"], s.rms_eps)
    qkv = n @ L["wqkv"].T
    q = qkv[:, :Hq * d].reshape(B, Hq, d)
    k = qkv[:, Hq * d:(Hq + Hkv) * d].reshape(B, Hkv, d)
    v = qkv[:, (Hq + Hkv) * d:].reshape(B, Hkv, d)
    q = rmsnorm(q, L["q_norm"], s.rms_eps)
    k = rmsnorm(k, L["k_norm"], s.rms_eps)
    pos = st.t + np.arange(B)
    base = rope_base(s)
    q, k = rope(q, pos, base), rope(k, pos, base)
    valid = _views.window_valid(s, st.t) & _views.keeps(s, _views.DROP_WINDOW)
    has_summary = st.t > 0 and _views.learned_summary(s)
    nval = ([_views.pooled_valid(s, st.t, bank) for bank in range(2)]
            if _views.pooled_summary(s) else [])
    o = np.empty((B, Hq, d))
    for h in range(Hq):
        g = h // rep
        pooled = [(st.PK[bank][j, g, :n], st.PV[bank][j, g, :n]) for bank, n in enumerate(nval)]
        o[:, h] = block_attention(q[:, h], k[:, g], v[:, g], st.Kw[j, g], st.Vw[j, g],
                                  valid, None if G is None else G[j, h], st.M[j, h],
                                  has_summary, pooled)
    x = x + o.reshape(B, Hq * d) @ L["wo"].T
    n2 = rmsnorm(x, L["post_norm"], s.rms_eps)
    gu = n2 @ L["w_gate_up"].T
    act = silu(gu[:, :s.mlp]) * gu[:, s.mlp:]
    return x + act @ L["w_down"].T


def forward(s, Wt, st: _views.ViewState, G, anchor, vocab_idx=None, trace=None):
    """Base logits z^(0) [B][V] (or [B][len(vocab_idx)] for a vocabulary
    sample) of one sequence. Wt: float64 weight dict (synth layout),
    st: that sequence's views, G: [D][Hq][R][d], anchor: the committed token.
    `trace`, if a dict, receives c, the slot inputs and every layer output.
    A drafter without the boundary view (ablation variant) has c = 0; one
    without the window or the summary attends to the other sources only."""
    if _views.keeps(s, _views.DROP_BOUNDARY):
        c = boundary_fusion(s, Wt, st.h)
    else:
        c = np.zeros(s.hidden)
    x = slot_init(s, Wt, c, int(anchor))
    if trace is not None:
        trace["c"], trace["x0"] = c, x.copy()
    for j in range(s.n_layers):
        x = layer(s, Wt["layers"][j], x, st, G, j)
        if trace is not None:
            trace[f"x{j + 1}"] = x.copy()
    n = rmsnorm(x, Wt["final_norm"], s.rms_eps)
    lm = Wt["lm_head"] if vocab_idx is None else Wt["lm_head"][vocab_idx]
    return n @ lm.T
