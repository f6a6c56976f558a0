"""Oracle for the fixed-size context views (Sec. 2.2; App. A.2, Eq. 10-11).

Per sequence the views are:

* the recent K/V window: the last min(t, W) target K/V rows of every selected
  layer, row p kept in ring slot p mod W (Sec. 2.2, App. B.1);
* the global summary: for every layer j, query head h and summary query
  r < R, the value m and log-normalizer eta of attention from the fixed query
  G[j,h,r] over all t target rows of the head's K/V group (Eq. 5, Eq. 10);
* the boundary hidden states h of the selected layers at the last ingested
  position (Sec. 2.2, the input of the boundary fusion).

The mean-pooled summary (the views as the configurations word them: strided
means instead of learned queries) replaces the learned summary when the shape
sets pool_slots: for each of two strides S, a ring of P slots in which slot
c mod P holds the mean K row and mean V row of chunk c = rows [cS, (c+1)S) of
every layer's K/V group, the open chunk with the mean of the rows it has so
far. A mean is the learned-query statistics of Eq. 10 with G = 0 (all scores
equal: uniform weights, eta = log of the count), merged chunk by chunk.

All arithmetic is float64. Inputs are float64 arrays holding the values of
the drawn tensors (bf16 values are exact in float64).
"""
from __future__ import annotations

import dataclasses

import numpy as np
import scipy.special


@dataclasses.dataclass
class ViewState:
    t: int            # target rows ingested so far (positions 0..t-1 cached)
    Kw: np.ndarray    # [D][Hkv][W][d]  window keys, slot = position mod W
    Vw: np.ndarray    # [D][Hkv][W][d]  window values
    M: np.ndarray     # [D][Hq][R][d]   summary values m
    eta: np.ndarray   # [D][Hq][R]      summary log-normalizers (-inf = empty)
    h: np.ndarray     # [L_b][hidden]   boundary hidden states
    PK: np.ndarray = None   # [2][D][Hkv][P][d] pooled key means (mean-pooled summary)
    PV: np.ndarray = None   # [2][D][Hkv][P][d] pooled value means
    SK: np.ndarray = None   # [2][D][Hkv][d]    sums of the open chunk's keys
    SV: np.ndarray = None   # [2][D][Hkv][d]    sums of the open chunk's values

    def copy(self) -> "ViewState":
        cp = lambda a: None if a is None else a.copy()
        return ViewState(self.t, self.Kw.copy(), self.Vw.copy(), self.M.copy(),
                         self.eta.copy(), self.h.copy(), cp(self.PK), cp(self.PV),
                         cp(self.SK), cp(self.SV))


def empty(s) -> ViewState:
    """The state before any row: t = 0, empty summary (eta = -inf, m = 0),
    zero window and boundary. Merging anything into it gives that thing
    (App. A.2: the merge is defined for nonempty sets; the empty set is its
    identity)."""
    D, Hq, Hkv, W, R, d = (s.n_layers, s.n_q_heads, s.n_kv_heads, s.window,
                           s.summary, s.head_dim)
    P = pool_slots(s)
    return ViewState(
        t=0,
        Kw=np.zeros((D, Hkv, W, d)), Vw=np.zeros((D, Hkv, W, d)),
        M=np.zeros((D, Hq, R, d)), eta=np.full((D, Hq, R), -np.inf),
        h=np.zeros((s.n_feat_layers, s.hidden)),
        PK=np.zeros((2, D, Hkv, P, d)), PV=np.zeros((2, D, Hkv, P, d)),
        SK=np.zeros((2, D, Hkv, d)), SV=np.zeros((2, D, Hkv, d)),
    )


def set_statistics(G, K, V, d):
    """eta_N and m_N of Eq. 10 for one head: G [R][d] queries, K/V [n][d]
    rows of the set N (n >= 1). Log-sum-exp with max subtraction (App. A.2)."""
    s = (G @ K.T) / np.sqrt(d)                    # s_j = g^T k_j / sqrt(d)   [R][n]
    mx = s.max(axis=1, keepdims=True)
    w = np.exp(s - mx)
    eta = mx[:, 0] + np.log(w.sum(axis=1))        # log sum_j exp(s_j)
    m = np.exp(s - eta[:, None]) @ V              # sum_j exp(s_j - eta) v_j
    return eta, m


def merge(eta_a, m_a, eta_n, m_n):
    """Eq. 11 with max subtraction: eta = log(e^eta_A + e^eta_N),
    m = e^(eta_A - eta) m_A + e^(eta_N - eta) m_N. An empty A (eta_A = -inf)
    returns N unchanged."""
    out_eta = np.empty_like(eta_n)
    out_m = np.empty_like(m_n)
    empty_a = np.isneginf(eta_a)
    out_eta[empty_a] = eta_n[empty_a]
    out_m[empty_a] = m_n[empty_a]
    f = ~empty_a
    mu = np.maximum(eta_a[f], eta_n[f])
    eta = mu + np.log(np.exp(eta_a[f] - mu) + np.exp(eta_n[f] - mu))
    out_eta[f] = eta
    out_m[f] = (np.exp(eta_a[f] - eta)[:, None] * m_a[f]
                + np.exp(eta_n[f] - eta)[:, None] * m_n[f])
    return out_eta, out_m


# Ablation variants (Sec. 3.4, Fig. "ablation"; App. D.3): a drafter built
# without one of the three views neither keeps nor reads it. Bits of
# `drop_views` in the shape:
DROP_WINDOW, DROP_SUMMARY, DROP_BOUNDARY = 1, 2, 4


def keeps(s, bit) -> bool:
    """Whether the shape's drafter keeps the view `bit`."""
    return not (getattr(s, "drop_views", 0) & bit)


def pool_slots(s) -> int:
    """P of the mean-pooled summary, 0 for the learned summary."""
    return int(getattr(s, "pool_slots", 0) or 0)


def learned_summary(s) -> bool:
    return keeps(s, DROP_SUMMARY) and pool_slots(s) == 0


def pooled_summary(s) -> bool:
    return keeps(s, DROP_SUMMARY) and pool_slots(s) > 0


def pooled_valid(s, t: int, bank: int) -> int:
    """Valid slots of a bank after t rows: the chunks begun so far, at most P
    (they fill slots 0, 1, ... before the ring wraps)."""
    S = s.pool_strides[bank]
    return min(-(-t // S), pool_slots(s))


def update(s, st: ViewState, G, K_new, V_new, h_new) -> ViewState:
    """Ingest n new target rows (Sec. 2.4, Inference; App. A.2).

    K_new, V_new: [n][D][Hkv][d] rows for positions t..t+n-1. h_new:
    [L_b][hidden] boundary states at the new boundary. n = 0 returns the
    state unchanged, h included (no row was committed, the boundary did not
    move). A dropped view (ablation variants) stays as `empty` made it."""
    n = K_new.shape[0]
    out = st.copy()
    if n == 0:
        return out
    W, d = s.window, s.head_dim
    rep = s.n_q_heads // s.n_kv_heads
    if keeps(s, DROP_WINDOW):
        for r in range(n):                          # ring write, in order
            out.Kw[:, :, (st.t + r) % W, :] = K_new[r]
            out.Vw[:, :, (st.t + r) % W, :] = V_new[r]
    if pooled_summary(s):
        P = pool_slots(s)
        for bank, S in enumerate(s.pool_strides):
            for r in range(n):                      # running mean of each chunk, in order
                p = st.t + r
                if p % S == 0:                      # a new chunk opens its slot
                    out.SK[bank] = 0.0
                    out.SV[bank] = 0.0
                out.SK[bank] += K_new[r]
                out.SV[bank] += V_new[r]
                k = (p // S) % P
                out.PK[bank][:, :, k] = out.SK[bank] / (p % S + 1)
                out.PV[bank][:, :, k] = out.SV[bank] / (p % S + 1)
    if learned_summary(s):
        for j in range(s.n_layers):
            for h in range(s.n_q_heads):
                g = h // rep                        # the head's K/V group
                eta_n, m_n = set_statistics(G[j, h], K_new[:, j, g, :], V_new[:, j, g, :], d)
                out.eta[j, h], out.M[j, h] = merge(st.eta[j, h], st.M[j, h], eta_n, m_n)
    if keeps(s, DROP_BOUNDARY):
        out.h = np.array(h_new, dtype=np.float64, copy=True)
    out.t = st.t + n
    return out


def brute_summary(s, G, K_all, V_all):
    """Eq. 5 directly: M = Attn(G, K_{1:t}, V_{1:t}) and its log-normalizer,
    for every layer and query head, over all t rows at once."""
    t = K_all.shape[0]
    D, Hq = s.n_layers, s.n_q_heads
    rep = Hq // s.n_kv_heads
    M = np.zeros((D, Hq, s.summary, s.head_dim))
    eta = np.full((D, Hq, s.summary), -np.inf)
    if t == 0:
        return M, eta
    for j in range(D):
        for h in range(Hq):
            K = K_all[:, j, h // rep, :]
            V = V_all[:, j, h // rep, :]
            sc = G[j, h] @ K.T / np.sqrt(s.head_dim)
            M[j, h] = scipy.special.softmax(sc, axis=1) @ V
            eta[j, h] = scipy.special.logsumexp(sc, axis=1)
    return M, eta


def brute_pooled(s, K_all, V_all):
    """Each bank's slots from the whole prefix at once: slot c mod P holds the
    mean of the rows of chunk c, for the last P chunks begun."""
    t = K_all.shape[0]
    P = pool_slots(s)
    PK = np.zeros((2, s.n_layers, s.n_kv_heads, P, s.head_dim))
    PV = np.zeros_like(PK)
    for bank, S in enumerate(s.pool_strides):
        C = -(-t // S)                              # chunks begun
        for c in range(max(0, C - P), C):
            rows = slice(c * S, min((c + 1) * S, t))
            PK[bank][:, :, c % P] = K_all[rows].mean(axis=0)
            PV[bank][:, :, c % P] = V_all[rows].mean(axis=0)
    return PK, PV


def brute_window(s, K_all, V_all):
    """The last min(t, W) rows, each at slot position mod W, and the mask of
    valid slots."""
    t = K_all.shape[0]
    W = s.window
    Kw = np.zeros((s.n_layers, s.n_kv_heads, W, s.head_dim))
    Vw = np.zeros_like(Kw)
    valid = np.zeros(W, dtype=bool)
    for p in range(max(0, t - W), t):
        Kw[:, :, p % W, :] = K_all[p]
        Vw[:, :, p % W, :] = V_all[p]
        valid[p % W] = True
    return Kw, Vw, valid


def window_valid(s, t: int) -> np.ndarray:
    """Slots holding a cached row after t rows: all W once t >= W, else 0..t-1."""
    valid = np.zeros(s.window, dtype=bool)
    valid[:min(t, s.window)] = True
    return valid


def state_bytes(s) -> int:
    """Bytes of one sequence's views as stored: window K and V in the model
    dtype, summary m and eta in fp32 per query head, boundary h in the model
    dtype. No term depends on t (Sec. 2.4, Fixed-cost complexity)."""
    el = 2 if s.dtype == "bf16" else 4
    window = 2 * s.n_layers * s.window * s.n_kv_heads * s.head_dim * el
    summary = s.n_layers * s.n_q_heads * s.summary * (s.head_dim + 1) * 4
    if pool_slots(s):   # two banks of P key and value means, fp32 sums of the open chunks
        summary = 2 * s.n_layers * s.n_kv_heads * s.head_dim * (
            2 * pool_slots(s) * el + 2 * 4)
    boundary = s.n_feat_layers * s.hidden * el
    return (window * keeps(s, DROP_WINDOW) + summary * keeps(s, DROP_SUMMARY) +
            boundary * keeps(s, DROP_BOUNDARY))
