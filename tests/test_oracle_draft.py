"""Pins of the drafter-forward oracle (Eq. 4, Eq. 6, Sec. 2.3, App. A.1,
App. B.1): library routines (torch rms_norm, scaled_dot_product_attention,
silu), an independent complex-number statement of RoPE, the LSE merge of
per-source attentions, a loop-by-loop brute force of the whole forward on a
micro shape, and structural invariants (GQA duplication, window order)."""
import math

import numpy as np
import pytest
import torch

import synth
from oracle import draft as Dr
from oracle import views as V

MICRO = synth.TINY.replace(name="micro", hidden=12, n_q_heads=4, n_kv_heads=2, head_dim=4,
                           mlp=10, vocab=17, n_layers=2, n_feat_layers=3, block=3,
                           window=5, summary=2, rope_theta=10000.0, ntk_alpha=2.0)


def rand_weights(s, seed, gain_std=0.3):
    w = synth.make_weights(s, seed=seed, std=0.3, gain_std=gain_std)
    return synth.weights_f64(w)


def rand_state(s, t, seed):
    rng = np.random.default_rng(seed)
    G = rng.normal(0, 1 / math.sqrt(s.head_dim), (s.n_layers, s.n_q_heads, s.summary,
                                                    s.head_dim))
    st = V.empty(s)
    if t:
        K = rng.normal(size=(t, s.n_layers, s.n_kv_heads, s.head_dim))
        Vv = rng.normal(size=K.shape)
        st = V.update(s, st, G, K, Vv, rng.normal(size=(s.n_feat_layers, s.hidden)))
    return st, G


def test_rmsnorm_matches_torch():
    x = np.random.default_rng(0).normal(size=(7, 33))
    g = np.random.default_rng(1).normal(size=33)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(x), (33,), torch.from_numpy(g), 1e-6)
    np.testing.assert_allclose(Dr.rmsnorm(x, g, 1e-6), ref.numpy(), rtol=1e-13)


def test_silu_matches_torch():
    x = np.linspace(-30, 30, 1001)
    np.testing.assert_allclose(Dr.silu(x), torch.nn.functional.silu(torch.from_numpy(x)).numpy(),
                               rtol=1e-13, atol=1e-300)


def test_rope_is_a_complex_rotation_of_half_pairs():
    rng = np.random.default_rng(2)
    d, base = 16, 5e5
    x = rng.normal(size=(6, 3, d))
    pos = np.array([0, 1, 7, 255, 4096, 262143])
    got = Dr.rope(x, pos, base)
    # independent statement: z_e = x_e + i x_{e+d/2}; z_e * exp(i pos / base^(2e/d))
    z = x[..., :d // 2] + 1j * x[..., d // 2:]
    theta = np.array([[p / base ** (2 * e / d) for e in range(d // 2)] for p in pos])
    zr = z * np.exp(1j * theta)[:, None, :]
    # angles near 2.6e5 rad carry ~1e-11 rad of rounding in either statement
    np.testing.assert_allclose(got, np.concatenate([zr.real, zr.imag], axis=-1), rtol=0,
                               atol=1e-10)
    np.testing.assert_array_equal(Dr.rope(x, np.zeros(6), base), x)   # position 0: identity


def _freqs(base, d):
    """Rotation frequency of every half pair, read off the oracle's rope: the
    angle of pair e at position 1 (a unit vector rotated once)."""
    x = np.zeros((1, 1, d))
    x[..., :d // 2] = 1.0
    y = Dr.rope(x, np.array([1]), base)
    return np.arctan2(y[0, 0, d // 2:], y[0, 0, :d // 2])


@pytest.mark.parametrize("d,alpha", [(4, 2.0), (64, 4.0), (128, 4.0), (128, 8.0)])
def test_rope_base_ntk_scales_the_lowest_frequency_by_alpha(d, alpha):
    """Fixed NTK scaling by alpha stretches the wavelength of the lowest
    rotary frequency by exactly alpha and leaves the highest (pair 0, one
    radian per position) unchanged, with the frequencies between still
    geometric; plain theta at alpha = 1."""
    s = MICRO.replace(head_dim=d, rope_theta=1e6, ntk_alpha=alpha)
    f1 = _freqs(Dr.rope_base(s.replace(ntk_alpha=1.0)), d)
    fa = _freqs(Dr.rope_base(s), d)
    assert Dr.rope_base(s.replace(ntk_alpha=1.0)) == 1e6
    assert fa[0] == pytest.approx(1.0, rel=1e-15) and f1[0] == pytest.approx(1.0, rel=1e-15)
    assert f1[-1] / fa[-1] == pytest.approx(alpha, rel=1e-9)
    np.testing.assert_allclose(fa[1:] / fa[:-1], fa[1] / fa[0], rtol=1e-9)


def test_boundary_fusion_closed_forms():
    """c = RMSNorm(W_fc [h_0; ...; h_{L_b-1}]): zero boundary states give
    c = 0; a unit entry k of feature layer l picks column l * hidden + k of
    W_fc (layer-major concatenation, [out][in] weights); a hand-computed
    2-wide case."""
    s = MICRO
    Wt = rand_weights(s, 31)
    h = np.zeros((s.n_feat_layers, s.hidden))
    assert np.array_equal(Dr.boundary_fusion(s, Wt, h), np.zeros(s.hidden))
    for l, k in ((0, 0), (1, 5), (2, 11)):
        h = np.zeros((s.n_feat_layers, s.hidden))
        h[l, k] = 1.0
        col = Wt["fc_w"][:, l * s.hidden + k]
        ref = col / np.sqrt(np.mean(col ** 2) + s.rms_eps) * Wt["fc_norm"]
        np.testing.assert_allclose(Dr.boundary_fusion(s, Wt, h), ref, rtol=1e-14)
    s2 = MICRO.replace(hidden=2, n_feat_layers=1, rms_eps=0.0)
    W2 = {"fc_w": np.array([[3.0, 0.0], [0.0, 4.0]]), "fc_norm": np.array([1.0, 2.0])}
    c = Dr.boundary_fusion(s2, W2, np.array([[1.0, 1.0]]))   # y = (3, 4), rms = sqrt(12.5)
    np.testing.assert_allclose(c, [3 / math.sqrt(12.5), 8 / math.sqrt(12.5)], rtol=1e-15)


def test_slot_init_closed_forms():
    """x_i = E[u_i] + P_i + c: slot 0 holds the anchor's embedding, slots
    1 .. B-1 the mask embedding; with E = 0 and c = 0 the slots are the
    positional encodings alone."""
    s = MICRO
    Wt = rand_weights(s, 32)
    zero_c = np.zeros(s.hidden)
    W0 = dict(Wt)
    W0["pos_emb"] = np.zeros_like(Wt["pos_emb"])
    x = Dr.slot_init(s, W0, zero_c, 9)
    assert np.array_equal(x[0], Wt["embed"][9])
    assert all(np.array_equal(x[i], Wt["mask_emb"]) for i in range(1, s.block))
    W1 = dict(Wt)
    W1["embed"] = np.zeros_like(Wt["embed"])
    W1["mask_emb"] = np.zeros_like(Wt["mask_emb"])
    assert np.array_equal(Dr.slot_init(s, W1, zero_c, 3), Wt["pos_emb"])
    c = np.arange(s.hidden, dtype=np.float64)
    assert np.array_equal(Dr.slot_init(s, W1, c, 3), Wt["pos_emb"] + c)


def test_positional_slots_reach_the_head_through_pass_through_layers():
    """Zero boundary states (c = 0), zero embeddings and layers whose output
    maps are zero: the logits are RMSNorm(P_i) W_lm^T, one row per slot."""
    s = MICRO
    Wt = rand_weights(s, 33)
    Wt["embed"] = np.zeros_like(Wt["embed"])
    Wt["mask_emb"] = np.zeros_like(Wt["mask_emb"])
    for L in Wt["layers"]:
        L["wo"][:] = 0
        L["w_down"][:] = 0
    st, G = rand_state(s, 6, 34)
    st.h[:] = 0.0
    ref = Dr.rmsnorm(Wt["pos_emb"], Wt["final_norm"], s.rms_eps) @ Wt["lm_head"].T
    np.testing.assert_allclose(Dr.forward(s, Wt, st, G, 4), ref, rtol=1e-13)


def test_block_attention_is_sdpa_over_the_concatenation():
    rng = np.random.default_rng(3)
    B, W, R, d = 5, 9, 4, 8
    q, kb, vb = (rng.normal(size=(B, d)) for _ in range(3))
    Kw, Vw = rng.normal(size=(W, d)), rng.normal(size=(W, d))
    G, M = rng.normal(size=(R, d)), rng.normal(size=(R, d))
    valid = np.array([1, 1, 0, 1, 0, 1, 1, 1, 0], dtype=bool)
    got = Dr.block_attention(q, kb, vb, Kw, Vw, valid, G, M, True)
    K = np.concatenate([kb, Kw, G])
    Vv = np.concatenate([vb, Vw, M])
    mask = torch.from_numpy(np.concatenate([np.ones(B, bool), valid, np.ones(R, bool)]))
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q)[None], torch.from_numpy(K)[None], torch.from_numpy(Vv)[None],
        attn_mask=mask[None, None, :].expand(1, B, -1))[0]
    np.testing.assert_allclose(got, ref.numpy(), rtol=1e-12, atol=1e-13)


def test_one_softmax_equals_merge_of_per_source_attentions():
    # one normalisation across three sources == Eq. 11 merge of the three partial attentions
    rng = np.random.default_rng(4)
    d = 8
    q = rng.normal(size=(1, d))
    parts = [(rng.normal(size=(n, d)), rng.normal(size=(n, d))) for n in (3, 6, 2)]
    got = Dr.block_attention(q, *parts[0], parts[1][0], parts[1][1], np.ones(6, bool),
                             parts[2][0], parts[2][1], True)
    eta, m = None, None
    for K, Vv in parts:
        e_n, m_n = V.set_statistics(q, K, Vv, d)
        if eta is None:
            eta, m = e_n, m_n
        else:
            eta, m = V.merge(eta, m, e_n, m_n)
    np.testing.assert_allclose(got, m, rtol=1e-13)


def test_single_key_attention_returns_the_value():
    rng = np.random.default_rng(5)
    q, kb, vb = (rng.normal(size=(1, 6)) for _ in range(3))
    out = Dr.block_attention(q, kb, vb, np.zeros((4, 6)), np.zeros((4, 6)), np.zeros(4, bool),
                             np.zeros((2, 6)), np.zeros((2, 6)), False)
    assert np.array_equal(out, vb)


# ---- brute force of the whole forward, written with scalar loops ----------------------------

def _loop_rms(x, g, eps):
    ms = sum(v * v for v in x) / len(x)
    return [v / math.sqrt(ms + eps) * gg for v, gg in zip(x, g)]


def _loop_matvec(Wm, x):            # Wm [out][in] (nn.Linear), y_o = sum_i W[o][i] x[i]
    return [sum(Wm[o][i] * x[i] for i in range(len(x))) for o in range(len(Wm))]


def brute_forward(s, Wt, st, G, a, no_window=False, no_summary=False, no_boundary=False,
                  pooled=None):
    """The whole forward with scalar loops; the flags leave a view's source out
    (ablation variants), whatever `st` holds for it. `pooled`: per bank, the
    (keys, values) [D][Hkv][n][d] of the valid slots of a mean-pooled summary,
    which then takes the learned summary's place."""
    B, H, Hk, d, hid = s.block, s.n_q_heads, s.n_kv_heads, s.head_dim, s.hidden
    base = s.rope_theta * s.ntk_alpha ** (d / (d - 2))
    hcat = [v for l in range(s.n_feat_layers) for v in st.h[l]]
    c = _loop_rms(_loop_matvec(Wt["fc_w"], hcat), Wt["fc_norm"], s.rms_eps)
    if no_boundary:
        c = [0.0] * hid
    x = []
    for i in range(B):
        e = Wt["embed"][a] if i == 0 else Wt["mask_emb"]
        x.append([e[k] + Wt["pos_emb"][i][k] + c[k] for k in range(hid)])
    nvalid = 0 if no_window else min(st.t, s.window)
    for j in range(s.n_layers):
        L = Wt["layers"][j]
        q = [[None] * H for _ in range(B)]
        k = [[None] * Hk for _ in range(B)]
        v = [[None] * Hk for _ in range(B)]
        for i in range(B):
            y = _loop_matvec(L["wqkv"], _loop_rms(x[i], L["in_norm"], s.rms_eps))
            for h in range(H):
                q[i][h] = _loop_rms(y[h * d:(h + 1) * d], L["q_norm"], s.rms_eps)
            for g in range(Hk):
                k[i][g] = _loop_rms(y[(H + g) * d:(H + g + 1) * d], L["k_norm"], s.rms_eps)
                v[i][g] = y[(H + Hk + g) * d:(H + Hk + g + 1) * d]
            for vecs in (q[i], k[i]):
                for n_ in range(len(vecs)):
                    u = vecs[n_]
                    r = list(u)
                    for e in range(d // 2):
                        ang = (st.t + i) / base ** (2 * e / d)
                        r[e] = u[e] * math.cos(ang) - u[e + d // 2] * math.sin(ang)
                        r[e + d // 2] = u[e] * math.sin(ang) + u[e + d // 2] * math.cos(ang)
                    vecs[n_] = r
        for i in range(B):
            o = []
            for h in range(H):
                g = h // (H // Hk)
                keys = [k[b][g] for b in range(B)] + [list(st.Kw[j, g, p]) for p in range(nvalid)]
                vals = [v[b][g] for b in range(B)] + [list(st.Vw[j, g, p]) for p in range(nvalid)]
                if pooled is not None:
                    for PKb, PVb in pooled:
                        keys += [list(PKb[j, g, n_]) for n_ in range(PKb.shape[2])]
                        vals += [list(PVb[j, g, n_]) for n_ in range(PVb.shape[2])]
                elif st.t > 0 and not no_summary:
                    keys += [list(G[j, h, r]) for r in range(s.summary)]
                    vals += [list(st.M[j, h, r]) for r in range(s.summary)]
                sc = [sum(q[i][h][e] * kk[e] for e in range(d)) / math.sqrt(d) for kk in keys]
                mx = max(sc)
                w = [math.exp(z - mx) for z in sc]
                tot = sum(w)
                o += [sum(w[n_] * vals[n_][e] for n_ in range(len(vals))) / tot for e in range(d)]
            x[i] = [a_ + b_ for a_, b_ in zip(x[i], _loop_matvec(L["wo"], o))]
        for i in range(B):
            n2 = _loop_rms(x[i], L["post_norm"], s.rms_eps)
            gu = _loop_matvec(L["w_gate_up"], n2)
            act = [gu[m] / (1 + math.exp(-gu[m])) * gu[s.mlp + m] for m in range(s.mlp)]
            x[i] = [a_ + b_ for a_, b_ in zip(x[i], _loop_matvec(L["w_down"], act))]
    return np.array([_loop_matvec(Wt["lm_head"], _loop_rms(x[i], Wt["final_norm"], s.rms_eps))
                     for i in range(B)])


@pytest.mark.parametrize("t", [0, 3, 5, 12])
def test_forward_matches_loop_brute_force(t):
    s = MICRO
    Wt = rand_weights(s, 11)
    st, G = rand_state(s, t, 12)
    got = Dr.forward(s, Wt, st, G, 6)
    ref = brute_forward(s, Wt, st, G, 6)
    assert got.shape == (s.block, s.vocab)
    np.testing.assert_allclose(got, ref, rtol=1e-10, atol=1e-11)


@pytest.mark.parametrize("drop", [1, 2, 4, 3, 6])
@pytest.mark.parametrize("t", [0, 3, 12])
def test_view_drop_variants_match_loop_brute_force(drop, t):
    """Ablation variants (Sec. 3.4, App. D.3): the variant's own update and
    forward equal the brute force over the full views with the dropped
    sources left out."""
    full = MICRO
    s = MICRO.replace(drop_views=drop)
    Wt = rand_weights(s, 11)
    st_full, G = rand_state(full, t, 12)
    st, _ = rand_state(s, t, 12)
    got = Dr.forward(s, Wt, st, G, 6)
    ref = brute_forward(full, Wt, st_full, G, 6, no_window=bool(drop & 1),
                        no_summary=bool(drop & 2), no_boundary=bool(drop & 4))
    np.testing.assert_allclose(got, ref, rtol=1e-10, atol=1e-11)
    if t:
        assert not np.allclose(got, Dr.forward(full, Wt, st_full, G, 6))


@pytest.mark.parametrize("t", [0, 1, 7, 12, 40])
def test_pooled_summary_forward_matches_loop_brute_force(t):
    """The mean-pooled summary's valid slots join the one softmax in place of
    the learned summary: the forward over the incrementally kept slots equals
    the loop brute force over slots recomputed from the whole prefix."""
    s = MICRO.replace(pool_strides=(2, 5), pool_slots=3)
    Wt = rand_weights(s, 31)
    rng = np.random.default_rng(32)
    K = rng.normal(size=(t, s.n_layers, s.n_kv_heads, s.head_dim))
    Vv = rng.normal(size=K.shape)
    st = V.empty(s)
    off = 0
    for n in (3, 1, 8, 2, 100):
        n = min(n, t - off)
        st = V.update(s, st, None, K[off:off + n], Vv[off:off + n],
                      np.ones((s.n_feat_layers, s.hidden)))
        off += n
    assert st.t == t
    PK, PV = V.brute_pooled(s, K, Vv)
    pooled = [(PK[b][:, :, :V.pooled_valid(s, t, b)], PV[b][:, :, :V.pooled_valid(s, t, b)])
              for b in range(2)]
    got = Dr.forward(s, Wt, st, None, 4)
    ref = brute_forward(s, Wt, st, None, 4, pooled=pooled)
    np.testing.assert_allclose(got, ref, rtol=1e-10, atol=1e-11)


def test_no_boundary_is_a_zero_fusion_weight():
    """c = RMSNorm(0) = 0: dropping the boundary view equals W_fc = 0."""
    s = MICRO.replace(drop_views=4)
    Wt = rand_weights(s, 21)
    st, G = rand_state(MICRO, 9, 22)
    W0 = dict(Wt)
    W0["fc_w"] = np.zeros_like(Wt["fc_w"])
    np.testing.assert_allclose(Dr.forward(s, Wt, st, G, 3), Dr.forward(MICRO, W0, st, G, 3),
                               rtol=1e-12, atol=1e-13)


def test_dropped_views_are_not_kept_and_do_not_count():
    """The variant keeps the other views exactly as the full drafter does, and
    its state bytes lose exactly the dropped view's term."""
    st_full, G = rand_state(MICRO, 9, 5)
    for drop in (1, 2, 4):
        s = MICRO.replace(drop_views=drop)
        st, _ = rand_state(s, 9, 5)
        assert st.t == st_full.t
        assert np.array_equal(st.Kw, st_full.Kw) != bool(drop & 1)
        assert np.array_equal(st.M, st_full.M) != bool(drop & 2)
        assert np.array_equal(st.h, st_full.h) != bool(drop & 4)
    el = 4
    win = 2 * MICRO.n_layers * MICRO.window * MICRO.n_kv_heads * MICRO.head_dim * el
    summ = MICRO.n_layers * MICRO.n_q_heads * MICRO.summary * (MICRO.head_dim + 1) * 4
    bnd = MICRO.n_feat_layers * MICRO.hidden * el
    assert V.state_bytes(MICRO) == win + summ + bnd
    assert V.state_bytes(MICRO.replace(drop_views=1)) == summ + bnd
    assert V.state_bytes(MICRO.replace(drop_views=2)) == win + bnd
    assert V.state_bytes(MICRO.replace(drop_views=4)) == win + summ


def test_gqa_equals_duplicated_kv_heads():
    s = MICRO                       # 4 q heads over 2 kv heads
    Wt = rand_weights(s, 13)
    st, G = rand_state(s, 9, 14)
    s2 = s.replace(n_kv_heads=4)    # every kv head duplicated for its two q heads
    Wt2 = {k: v for k, v in Wt.items()}
    Wt2["layers"] = []
    d, H = s.head_dim, s.n_q_heads
    for L in Wt["layers"]:
        q = L["wqkv"][:H * d]
        k = L["wqkv"][H * d:(H + 2) * d].reshape(2, d, -1)
        v = L["wqkv"][(H + 2) * d:].reshape(2, d, -1)
        L2 = dict(L)
        L2["wqkv"] = np.concatenate([q, np.repeat(k, 2, axis=0).reshape(4 * d, -1),
                                     np.repeat(v, 2, axis=0).reshape(4 * d, -1)])
        Wt2["layers"].append(L2)
    st2 = V.ViewState(st.t, np.repeat(st.Kw, 2, axis=1), np.repeat(st.Vw, 2, axis=1), st.M,
                      st.eta, st.h)
    np.testing.assert_allclose(Dr.forward(s, Wt, st, G, 3), Dr.forward(s2, Wt2, st2, G, 3),
                               rtol=1e-12, atol=1e-13)


def test_window_slot_order_does_not_matter():
    s = MICRO
    Wt = rand_weights(s, 15)
    st, G = rand_state(s, 23, 16)          # full window
    perm = np.random.default_rng(0).permutation(s.window)
    st2 = st.copy()
    st2.Kw, st2.Vw = st.Kw[:, :, perm], st.Vw[:, :, perm]
    np.testing.assert_allclose(Dr.forward(s, Wt, st, G, 1), Dr.forward(s, Wt, st2, G, 1),
                               rtol=1e-12, atol=1e-13)


def test_layers_with_zero_output_maps_pass_the_slots_through():
    s = MICRO
    Wt = rand_weights(s, 17)
    for L in Wt["layers"]:
        L["wo"][:] = 0
        L["w_down"][:] = 0
    st, G = rand_state(s, 7, 18)
    a = 5
    c = Dr.rmsnorm(Wt["fc_w"] @ st.h.reshape(-1), Wt["fc_norm"], s.rms_eps)
    x = np.stack([Wt["embed"][a]] + [Wt["mask_emb"]] * (s.block - 1)) + Wt["pos_emb"] + c
    ref = Dr.rmsnorm(x, Wt["final_norm"], s.rms_eps) @ Wt["lm_head"].T
    np.testing.assert_allclose(Dr.forward(s, Wt, st, G, a), ref, rtol=1e-13)


def test_vocab_sample_matches_full_logits():
    s = MICRO
    Wt = rand_weights(s, 19)
    st, G = rand_state(s, 4, 20)
    idx = np.array([16, 0, 5, 5, 9])
    np.testing.assert_allclose(Dr.forward(s, Wt, st, G, 2, vocab_idx=idx),
                               Dr.forward(s, Wt, st, G, 2)[:, idx], rtol=1e-13)
