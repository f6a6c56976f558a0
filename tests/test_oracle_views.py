"""Pins of the views oracle (Sec. 2.2; App. A.2 Eq. 10-11; Sec. 2.4) against
brute force over the whole prefix (Eq. 5), closed forms and the paper's
printed state sizes."""
import json
import os

import numpy as np
import pytest

import synth
from oracle import views as V

HERE = os.path.dirname(os.path.abspath(__file__))
# A small GQA shape (2 q heads per kv head) so that group indexing is exercised.
S = synth.TINY.replace(name="mini", hidden=64, n_q_heads=4, n_kv_heads=2, head_dim=16,
                       n_layers=2, n_feat_layers=2, window=8, summary=3, block=4,
                       vocab=50, mlp=96)


def rows(n, seed, scale=1.0):
    rng = np.random.default_rng(seed)
    shp = (n, S.n_layers, S.n_kv_heads, S.head_dim)
    return rng.normal(0, scale, shp), rng.normal(0, scale, shp)


def Gq(seed=1, scale=1.0):
    rng = np.random.default_rng(seed)
    return rng.normal(0, scale / np.sqrt(S.head_dim), (S.n_layers, S.n_q_heads, S.summary,
                                                       S.head_dim))


def ingest(G, K, Vv, sizes):
    st = V.empty(S)
    h = np.zeros((S.n_feat_layers, S.hidden))
    off = 0
    for n in sizes:
        st = V.update(S, st, G, K[off:off + n], Vv[off:off + n], h + off)
        off += n
    return st


@pytest.mark.parametrize("gscale", [1.0, 8.0, 60.0])
def test_incremental_equals_brute_force(gscale):
    # init over a 40-row prefix, then 64 decode updates of 17 rows (Eq. 5 vs Eq. 11)
    G = Gq(scale=gscale)
    sizes = [40] + [17] * 64
    K, Vv = rows(sum(sizes), 2)
    st = ingest(G, K, Vv, sizes)
    M, eta = V.brute_summary(S, G, K, Vv)
    assert st.t == sum(sizes)
    np.testing.assert_allclose(st.M, M, rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(st.eta, eta, rtol=1e-12, atol=1e-12)


def test_chunking_and_order_invariance():
    G = Gq()
    K, Vv = rows(300, 3)
    a = ingest(G, K, Vv, [300])
    b = ingest(G, K, Vv, [1] * 8 + [100, 0, 17, 175])
    np.testing.assert_allclose(a.M, b.M, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(a.eta, b.eta, rtol=1e-13)
    perm = np.random.default_rng(0).permutation(300)
    c = ingest(G, K[perm], Vv[perm], [300])          # the summary is a set function
    np.testing.assert_allclose(a.M, c.M, rtol=1e-12, atol=1e-13)


def test_single_key_returns_value_exactly():
    G = Gq()
    K, Vv = rows(1, 4)
    st = ingest(G, K, Vv, [1])
    rep = S.n_q_heads // S.n_kv_heads
    for j in range(S.n_layers):
        for h in range(S.n_q_heads):
            for r in range(S.summary):
                assert np.array_equal(st.M[j, h, r], Vv[0, j, h // rep])
                s = G[j, h, r] @ K[0, j, h // rep] / np.sqrt(S.head_dim)
                assert st.eta[j, h, r] == pytest.approx(s, rel=1e-15)


def test_constant_values_pool_to_the_constant():
    G = Gq(scale=5.0)
    K, _ = rows(200, 5)
    c = np.random.default_rng(6).normal(size=(S.n_layers, S.n_kv_heads, S.head_dim))
    Vv = np.broadcast_to(c, K.shape).copy()
    st = ingest(G, K, Vv, [50, 17, 17, 116])
    rep = S.n_q_heads // S.n_kv_heads
    for h in range(S.n_q_heads):
        np.testing.assert_allclose(st.M[:, h], np.broadcast_to(c[:, h // rep, None, :],
                                                                st.M[:, h].shape), rtol=1e-13)


def test_zero_queries_give_the_mean():
    G = np.zeros((S.n_layers, S.n_q_heads, S.summary, S.head_dim))
    K, Vv = rows(123, 7)
    st = ingest(G, K, Vv, [23, 100])
    rep = S.n_q_heads // S.n_kv_heads
    for j in range(S.n_layers):
        for h in range(S.n_q_heads):
            np.testing.assert_allclose(st.M[j, h], np.broadcast_to(
                Vv[:, j, h // rep].mean(axis=0), st.M[j, h].shape), rtol=1e-12)
            np.testing.assert_allclose(st.eta[j, h], np.log(123.0), rtol=1e-14)


def test_empty_update_is_identity():
    G = Gq()
    K, Vv = rows(30, 8)
    st = ingest(G, K, Vv, [30])
    e = V.update(S, st, G, K[:0], Vv[:0], np.ones((S.n_feat_layers, S.hidden)))
    for f in ("Kw", "Vw", "M", "eta", "h"):
        assert np.array_equal(getattr(st, f), getattr(e, f))
    assert e.t == st.t
    z = V.empty(S)                                   # and on the empty state
    e0 = V.update(S, z, G, K[:0], Vv[:0], np.ones((S.n_feat_layers, S.hidden)))
    assert np.all(np.isneginf(e0.eta)) and e0.t == 0


@pytest.mark.parametrize("sizes", [[3], [8], [5, 3], [5, 4], [7, 17, 17, 2], [30], [0, 9, 0],
                                   [1] * 19])
def test_window_is_the_last_rows(sizes):
    G = Gq()
    K, Vv = rows(sum(sizes), 9)
    st = ingest(G, K, Vv, sizes)
    Kw, Vw, valid = V.brute_window(S, K, Vv)
    assert np.array_equal(valid, V.window_valid(S, st.t))
    assert np.array_equal(st.Kw[:, :, valid], Kw[:, :, valid])
    assert np.array_equal(st.Vw[:, :, valid], Vw[:, :, valid])


def test_boundary_state_follows_the_last_update():
    G = Gq()
    K, Vv = rows(10, 10)
    st = ingest(G, K, Vv, [4, 6])
    assert np.array_equal(st.h, np.zeros((S.n_feat_layers, S.hidden)) + 4)


def test_state_bytes_reproduce_the_papers_numbers():
    with open(os.path.join(HERE, "golden", "state_size.json")) as f:
        gold = json.load(f)
    MiB = 2 ** 20
    s8 = synth.QWEN3_8B
    # DSpark keeps K and V of every token for the 5 selected layers (bf16, 8 kv heads)
    per_token = 2 * s8.n_layers * s8.n_kv_heads * s8.head_dim * 2
    assert per_token * 32768 / MiB == gold["dspark_mib_at_32k"]
    assert per_token * 131072 / MiB == gold["dspark_mib_at_128k"]
    b = V.state_bytes(s8)
    assert b == 6_604_800
    assert round(b / MiB, 1) == gold["longspark_mib"]
    assert round(gold["dspark_mib_at_128k"] * MiB / b) == gold["reduction_at_128k"]
    assert V.state_bytes(synth.QWEN3_32B) == 7_936_000
    assert V.state_bytes(synth.TINY) == 150_784


# ---- the mean-pooled summary (the views as the configurations word them) --------------------

SP = S.replace(name="mini-pooled", pool_strides=(3, 8), pool_slots=4)


def ingest_pooled(K, Vv, sizes, s=SP):
    st = V.empty(s)
    h = np.zeros((s.n_feat_layers, s.hidden))
    off = 0
    for n in sizes:
        st = V.update(s, st, None, K[off:off + n], Vv[off:off + n], h + off)
        off += n
    return st


@pytest.mark.parametrize("sizes", [[1] * 70, [40] + [17] * 5, [2, 5, 1, 31, 3, 9, 100],
                                   [0, 3, 0, 1], [24], [23, 1, 8]])
def test_pooled_incremental_equals_brute_force(sizes):
    """Slot c mod P of each bank holds the mean of chunk c's rows, for the last
    P chunks begun, however the rows arrive (chunks and the ring cross updates)."""
    t = sum(sizes)
    K, Vv = rows(t, 31)
    st = ingest_pooled(K, Vv, sizes)
    PK, PV = V.brute_pooled(SP, K, Vv)
    assert st.t == t
    np.testing.assert_allclose(st.PK, PK, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(st.PV, PV, rtol=1e-12, atol=1e-12)
    for bank, S_ in enumerate(SP.pool_strides):
        assert V.pooled_valid(SP, t, bank) == min(-(-t // S_), SP.pool_slots)
    # the learned summary is not kept
    assert np.all(st.M == 0) and np.all(np.isneginf(st.eta))


def test_pooled_slots_by_hand():
    """Stride 3, 4 slots, 14 rows of scalar-like values: chunk means by hand."""
    s = SP
    K = np.zeros((14, s.n_layers, s.n_kv_heads, s.head_dim))
    for p in range(14):
        K[p] = p
    st = ingest_pooled(K, -K, [5, 4, 5])
    # chunks of 3: [0,1,2] [3,4,5] [6,7,8] [9,10,11] [12,13]; 5 chunks > 4 slots
    want = {0: 12.5, 1: 4.0, 2: 7.0, 3: 10.0}       # slot 0 recycled by chunk 4
    for k, m in want.items():
        assert np.all(st.PK[0][:, :, k] == m) and np.all(st.PV[0][:, :, k] == -m)
    # stride 8: [0..7] mean 3.5, [8..13] mean 10.5 (open chunk)
    assert np.all(st.PK[1][:, :, 0] == 3.5) and np.all(st.PK[1][:, :, 1] == 10.5)
    assert V.pooled_valid(s, 14, 0) == 4 and V.pooled_valid(s, 14, 1) == 2


def test_pooled_constant_rows_pool_to_the_constant():
    K, Vv = rows(50, 3)
    K[:] = 0.625
    Vv[:] = -1.75
    st = ingest_pooled(K, Vv, [13, 20, 17])
    assert np.all(st.PK[:, :, :, :, :] == 0.625) and np.all(st.PV == -1.75)


def test_pooled_mean_is_the_zero_query_statistics():
    """A slot is Eq. 10 with G = 0: uniform weights give the mean, and the
    log-normaliser is the log of the chunk's row count."""
    K, Vv = rows(8, 4)
    st = ingest_pooled(K, Vv, [8])
    j, g = 1, 1
    eta, m = V.set_statistics(np.zeros((1, S.head_dim)), K[:, j, g], Vv[:, j, g], S.head_dim)
    np.testing.assert_allclose(m[0], st.PV[1][j, g, 0], rtol=1e-13)
    assert abs(eta[0] - np.log(8)) < 1e-13


def test_pooled_state_bytes_are_fixed():
    el = 4
    s = SP
    want = (2 * s.n_layers * s.window * s.n_kv_heads * s.head_dim * el
            + 2 * s.n_layers * s.n_kv_heads * s.head_dim * (2 * s.pool_slots * el + 8)
            + s.n_feat_layers * s.hidden * el)
    assert V.state_bytes(s) == want
    assert V.state_bytes(synth.TINY_POOLED) < V.state_bytes(synth.TINY_POOLED.replace(window=128))


def test_nan_in_a_key_row_stays_in_its_group_and_layer():
    """A NaN entry in the key of row p, layer j, group g: the window slot
    p mod W of (j, g) holds it until row p + W replaces it; the summary of
    the query heads reading group g in layer j becomes NaN and stays NaN (Eq. 5
    covers every row ever ingested); every other layer, group and head stays
    finite, and the boundary is untouched."""
    G = Gq()
    K, Vv = rows(30, 41)
    p, j, g = 5, 1, 0
    K[p, j, g, 3] = np.nan
    st = ingest(G, K[:9], Vv[:9], [4, 5])
    rep = S.n_q_heads // S.n_kv_heads
    heads = list(range(g * rep, (g + 1) * rep))
    assert np.isnan(st.Kw[j, g, p % S.window]).any()
    bad = np.zeros(st.Kw.shape, dtype=bool)
    bad[j, g, p % S.window] = True
    assert np.all(np.isfinite(st.Kw[~bad])) and np.all(np.isfinite(st.Vw))
    for jj in range(S.n_layers):
        for h in range(S.n_q_heads):
            nan = jj == j and h in heads
            assert np.isnan(st.eta[jj, h]).all() == nan
            assert np.isnan(st.M[jj, h]).all() == nan
            if not nan:
                assert np.all(np.isfinite(st.eta[jj, h])) and np.all(np.isfinite(st.M[jj, h]))
    assert np.all(np.isfinite(st.h))
    st2 = V.update(S, st, G, K[9:9 + S.window], Vv[9:9 + S.window],
                   np.zeros((S.n_feat_layers, S.hidden)))        # row p leaves the window
    assert np.all(np.isfinite(st2.Kw))
    assert np.isnan(st2.eta[j, heads]).all() and np.isnan(st2.M[j, heads]).all()


def test_inf_in_a_value_row_leaves_the_normalisers_finite():
    """eta depends on the keys alone (Eq. 10): an infinite value entry makes
    the summary values M of the heads reading it non-finite in that one
    coordinate, while every eta stays finite and equal to the clean run's."""
    G = Gq()
    K, Vv = rows(12, 43)
    clean = ingest(G, K, Vv, [7, 5])
    Vv[2, 0, 1, 6] = np.inf
    st = ingest(G, K, Vv, [7, 5])
    rep = S.n_q_heads // S.n_kv_heads
    np.testing.assert_array_equal(st.eta, clean.eta)
    for h in range(S.n_q_heads):
        hit = h // rep == 1
        assert (~np.isfinite(st.M[0, h, :, 6])).all() == hit
        other = np.delete(st.M[0, h], 6, axis=1) if hit else st.M[0, h]
        assert np.all(np.isfinite(other))
    np.testing.assert_array_equal(st.M[1], clean.M[1])
