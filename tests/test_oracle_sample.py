"""Pins of the sampler oracle (Eq. 8): Philox4x32-10 against its published
known-answer vectors, the fp32 logarithm against numpy's log, Gumbel moments
(closed forms), the two-level Gumbel-max against the one-level one in its two
degenerate cases (one chunk; one token per chunk), its frequencies against
softmax(z/T) (chi-square), greedy against numpy argmax, top-k support against
a sort, lse closed forms."""
import json
import math
import os

import numpy as np
import pytest
import scipy.stats

from oracle import sample as Sm
from oracle.sample import gumbel, proposal, sample, verify, verify_gumbel, verify_uniform


def test_philox_known_answers():
    """Philox4x32-10 against the generator's published known-answer vectors."""
    kat = json.load(open(os.path.join(os.path.dirname(__file__), "golden",
                                      "philox4x32_10_kat.json")))
    for vec in kat["vectors"]:
        ctr = [np.uint64(int(x, 16)) for x in vec["ctr"]]
        key = [np.uint64(int(x, 16)) for x in vec["key"]]
        got = [int(w) for w in Sm.philox4x32_10(ctr, key)]
        assert got == [int(x, 16) for x in vec["out"]]


def test_noise_counter_layout():
    """Token v of row r in stream s is word v mod 4 of the block of counter
    (v div 4, r, step mod 2^32, (step div 2^32) mod 2^30 + 2^30 s), key the
    seed's two halves."""
    seed, step = 0x123456789ABCDEF0, 0x0000000500000007
    for s_, r, v in ((0, 3, 10), (1, 0, 0), (2, 7, 4095)):
        w = Sm.philox4x32_10((np.uint64(v // 4), np.uint64(r), np.uint64(7),
                              np.uint64(5 | (s_ << 30))),
                             (np.uint64(0x9ABCDEF0), np.uint64(0x12345678)))
        assert int(Sm.philox_bits(seed, step, r, v, stream=s_)) == int(w[v % 4])


def test_logf_within_three_ulp_of_numpy():
    rng = np.random.default_rng(0)
    x = np.concatenate([
        rng.uniform(1e-7, 20.0, 400_000), np.exp(rng.uniform(-87, 88, 200_000)),
        2.0 ** np.arange(-126, 127), [np.nextafter(1.0, 0.0), 1.0, 1.4142135, 1.4142137,
                                      0.70710677, 5.9604645e-08, 16.635532]]).astype(np.float32)
    got = Sm.logf(x).astype(np.float64)
    ref = np.log(x.astype(np.float64))
    ulp = np.spacing(np.abs(ref).astype(np.float32)).astype(np.float64)
    ulp = np.maximum(ulp, np.spacing(np.float32(0)))
    assert np.max(np.abs(got - ref) / ulp) <= 3.0
    assert Sm.logf(np.float32([1.0]))[0] == 0.0


def test_uniform_is_exact_and_open():
    bits = np.array([0, 511, 512, 2 ** 31, 2 ** 32 - 1], dtype=np.uint32)
    u = Sm.uniform(bits)
    assert u[0] == 2.0 ** -24 and u[1] == 2.0 ** -24 and u[2] == 3 * 2.0 ** -24
    assert u[-1] == 1 - 2.0 ** -24
    assert np.all((u > 0) & (u < 1))


def test_gumbel_moments():
    g = Sm.gumbel(5, 0, np.arange(2000)[:, None], np.arange(1000)[None, :]).astype(np.float64)
    # standard Gumbel: mean = Euler-Mascheroni gamma, variance = pi^2 / 6
    assert abs(g.mean() - 0.5772156649) < 0.004
    assert abs(g.var() - math.pi ** 2 / 6) < 0.01
    assert np.isfinite(g).all() and g.max() < 16.7


def test_noise_streams_differ_by_seed_step_and_row():
    v = np.arange(64)
    a = Sm.philox_bits(1, 0, 0, v)
    assert len(set(a.tolist())) == 64
    for other in (Sm.philox_bits(2, 0, 0, v), Sm.philox_bits(1, 1, 0, v),
                  Sm.philox_bits(1, 0, 1, v), Sm.philox_bits(1, 0, 0, v, stream=2),
                  Sm.philox_bits(1, 2 ** 32, 0, v)):
        assert np.mean(a == other) < 0.05


@pytest.mark.parametrize("T,top_k", [(1.0, 0), (0.7, 0), (1.3, 3)])
def test_gumbel_max_frequencies_follow_softmax(T, top_k):
    z = np.float32([0.3, -1.2, 1.1, 0.0, 2.0, -0.4])
    n = 30_000
    y, _, _ = Sm.sample(np.tile(z, (n, 1)), T, top_k, 42, 7, rows_per_pass=4096)
    counts = np.bincount(y, minlength=6).astype(np.float64)
    S = Sm.support(z, top_k)
    zs = z[S].astype(np.float64) / T
    p = np.exp(zs - zs.max())
    p = p / p.sum()
    assert counts.sum() == counts[S].sum()
    chi2 = scipy.stats.chisquare(counts[S], p * n)
    assert chi2.pvalue > 1e-3


def test_logq_is_the_log_probability_of_the_token():
    z = np.float32([0.5, 1.5, -0.25, 3.0])
    T = float(np.float32(0.8))                  # the temperature is an fp32 argument
    y, lse, logq = Sm.sample_row(z, 0.8, 0, 1, 2, 3)
    assert lse == pytest.approx(math.log(sum(math.exp(float(v) / T) for v in z)), rel=1e-12)
    assert logq == pytest.approx(float(z[y]) / T - lse, rel=1e-12)
    # the empirical frequency of each token matches exp(log q)
    n = 20_000
    ys, _, lq = Sm.sample(np.tile(z, (n, 1)), 0.8, 0, 3, 4, rows_per_pass=4096)
    for v in range(4):
        sel = ys == v
        assert abs(sel.mean() - math.exp(lq[sel][0])) < 0.015


def test_lse_closed_forms():
    V = 1000
    z = np.full(V, np.float32(2.5))
    _, lse, logq = Sm.sample_row(z, 0.5, 0, 0, 0, 0)
    assert lse == pytest.approx(5.0 + math.log(V), rel=1e-13)
    assert logq == pytest.approx(-math.log(V), rel=1e-12)
    p = np.random.default_rng(1).dirichlet(np.ones(50))
    _, lse, _ = Sm.sample_row(np.log(p).astype(np.float32), 1.0, 0, 0, 0, 0)
    assert abs(lse) < 1e-6


def test_greedy_is_first_argmax():
    rng = np.random.default_rng(2)
    z = rng.normal(size=(50, 300)).astype(np.float32)
    z[3, [10, 200]] = 9.0                       # tie: the lower index wins
    y, lse, logq = Sm.sample(z, 0.0, 0, 0, 0)
    assert np.array_equal(y, np.argmax(z, axis=1))
    assert y[3] == 10 and np.all(logq == 0.0)


def test_top_k_support_is_the_k_largest_lower_index_first():
    z = np.float32([1.0, 3.0, 3.0, -2.0, 3.0, 0.5, 2.0])
    assert Sm.support(z, 2).tolist() == [1, 2]
    assert Sm.support(z, 4).tolist() == [1, 2, 4, 6]
    assert Sm.support(z, 0).tolist() == list(range(7))
    rng = np.random.default_rng(3)
    for _ in range(20):
        zz = rng.integers(-3, 3, 40).astype(np.float32)
        k = int(rng.integers(1, 40))
        brute = sorted(range(40), key=lambda v: (-float(zz[v]), v))[:k]
        assert Sm.support(zz, k).tolist() == sorted(brute)


def test_sampled_token_is_in_the_top_k_support():
    rng = np.random.default_rng(4)
    z = rng.normal(size=(40, 500)).astype(np.float32)
    y, _, _ = Sm.sample(z, 1.0, 5, 9, 1)
    for r in range(40):
        assert y[r] in set(Sm.support(z[r], 5).tolist())


# ---- the two-level draw --------------------------------------------------------------------

def test_one_chunk_is_the_flat_gumbel_max():
    """With one chunk over the whole vocabulary the draw is the one-level
    Gumbel-max: the first argmax of fl(fl(z/T) + g) with the token noise."""
    rng = np.random.default_rng(11)
    z = rng.normal(size=(30, 257)).astype(np.float32) * np.float32(2.0)
    for T in (1.0, 0.6):
        y, _, _ = Sm.sample(z, T, 0, 5, 8, chunk=257)
        zt = (z / np.float32(T)).astype(np.float32)
        for r in range(30):
            key = (zt[r] + Sm.gumbel(5, 8, r, np.arange(257))).astype(np.float32)
            assert y[r] == int(np.argmax(key))


def test_unit_chunks_draw_from_the_chunk_stream():
    """With one token per chunk, L_c = z_c/T exactly, so the draw is the
    one-level Gumbel-max with the chunk noise (stream 3) in place of the
    token noise."""
    rng = np.random.default_rng(12)
    z = rng.normal(size=(30, 100)).astype(np.float32) * np.float32(3.0)
    for T, k in ((1.0, 0), (0.8, 0), (1.0, 9)):
        y, _, _ = Sm.sample(z, T, k, 6, 2, chunk=1)
        zt = (z / np.float32(T)).astype(np.float32)
        for r in range(30):
            key = (zt[r] + Sm.gumbel(6, 2, r, np.arange(100), stream=3)).astype(np.float32)
            S = Sm.support(z[r], k)
            masked = np.full(100, -np.inf, dtype=np.float32)
            masked[S] = key[S]
            assert y[r] == int(np.argmax(masked))


def test_chunk_log_mass_brute_force():
    """L_c against a scalar loop over each chunk's support tokens, with a
    ragged last chunk and a chunk left empty by the support."""
    rng = np.random.default_rng(13)
    zt = rng.normal(size=(3, 37)) * 4.0
    inside = rng.random((3, 37)) < 0.6
    inside[1, 16:32] = False
    L = Sm.chunk_log_mass(zt, inside, 16)
    assert L.shape == (3, 3)
    for r in range(3):
        for c in range(3):
            terms = [math.exp(zt[r, v]) for v in range(16 * c, min(37, 16 * c + 16)) if inside[r, v]]
            if terms:
                assert L[r, c] == pytest.approx(math.log(sum(terms)), rel=1e-13, abs=1e-13)
            else:
                assert L[r, c] == -np.inf


@pytest.mark.parametrize("T,top_k", [(1.0, 0), (0.7, 0), (1.0, 11)])
def test_two_level_frequencies_follow_softmax(T, top_k):
    """Several chunks, the last ragged (V = 40 in chunks of 16), top-k
    supports that cut chunks: the token frequencies follow softmax(z/T) over
    the support (chi-square), and every token's log q is its log frequency."""
    z = np.float32([0.3, -1.2, 1.1, 0.0, 2.0, -0.4, 0.9, 1.4, -2.0, 0.5,
                    1.0, 1.0, -0.3, 0.2, 1.7, -1.1, 0.8, 0.1, 1.2, -0.6,
                    0.4, 1.9, -0.9, 0.6, 1.3, -1.5, 0.7, 0.0, 1.6, -0.2,
                    1.1, 0.3, -0.7, 1.8, 0.2, -1.3, 0.9, 1.5, -0.1, 1.0])
    n = 60_000
    y, _, lq = Sm.sample(np.tile(z, (n, 1)), T, top_k, 43, 9, rows_per_pass=4096)
    S = Sm.support(z, top_k)
    counts = np.bincount(y, minlength=40).astype(np.float64)
    assert counts.sum() == counts[S].sum()
    zs = z[S].astype(np.float64) / float(np.float32(T))
    p = np.exp(zs - zs.max())
    p = p / p.sum()
    assert scipy.stats.chisquare(counts[S], p * n).pvalue > 1e-3
    for v in S[:5]:
        sel = y == v
        assert abs(np.exp(lq[sel][0]) - p[list(S).index(v)]) < 1e-12


def test_chunk_choice_and_token_of_the_detail():
    """The reported chunk keys are fl(fl32(L_c) + h_c), the chosen chunk is
    their first argmax and the token lies in it."""
    rng = np.random.default_rng(14)
    z = rng.normal(size=(8, 100)).astype(np.float32)
    y, _, _, K, c = Sm.sample(z, 1.0, 0, 3, 1, detail=True)
    inside = np.ones(z.shape, dtype=bool)
    L = Sm.chunk_log_mass(z.astype(np.float64), inside)
    for r in range(8):
        h = Sm.gumbel(3, 1, r, np.arange(7), stream=3)
        assert np.array_equal(K[r], (L[r].astype(np.float32) + h).astype(np.float32))
        assert c[r] == int(np.argmax(K[r])) and y[r] // 16 == c[r]


# ---- Markov-corrected sampling (Eq. 7-8) ----------------------------------------------------

def _markov_inputs(nb, B, V, r, seed, scale=0.5):
    g = np.random.default_rng(seed)
    z0 = g.normal(size=(nb, B, V)).astype(np.float32)
    E = (g.normal(size=(V, r)) * scale).astype(np.float32)
    W = (g.normal(size=(V, r)) * scale).astype(np.float32)
    a = g.integers(0, V, size=nb)
    return z0, a, E, W


@pytest.mark.parametrize("T,top_k", [(1.0, 0), (0.6, 3), (0.0, 0)])
def test_markov_without_correction_is_the_plain_sampler(T, top_k):
    """W_c = 0: the corrected logits are the base logits and every output is
    the plain sampler's on the [batch * B][V] rows."""
    z0, a, E, W = _markov_inputs(5, 4, 37, 8, 1)
    y, lse, logq, z = Sm.sample_markov(z0, a, E, np.zeros_like(W), T, top_k, 11, 3)
    assert np.array_equal(z, z0)
    y1, lse1, logq1 = Sm.sample(z0.reshape(-1, 37), T, top_k, 11, 3)
    assert np.array_equal(y.reshape(-1), y1)
    assert np.array_equal(lse.reshape(-1), lse1) and np.array_equal(logq.reshape(-1), logq1)


def test_markov_correction_closed_form():
    """One-hot correction embeddings pick one column of W_c: c_v = W_c[v, y mod r]."""
    V, r = 12, 4
    E = np.zeros((V, r), dtype=np.float32)
    E[np.arange(V), np.arange(V) % r] = 1.0
    W = np.random.default_rng(2).normal(size=(V, r)).astype(np.float32)
    c = Sm.correction(E, W, [0, 5, 11])
    assert np.array_equal(c, W[:, [0, 1, 3]].T)



def test_markov_correction_is_exact_on_integer_values():
    """Small integers make every fp32 product and partial sum exact, so the
    ordered fp32 chain must equal the float64 product W_c E_c(y) exactly
    (a dropped term, a transposed operand or a wrong row would not)."""
    V, r = 37, 24
    g = np.random.default_rng(4)
    E = g.integers(-8, 9, size=(V, r)).astype(np.float32)
    W = g.integers(-8, 9, size=(V, r)).astype(np.float32)
    y = np.array([0, 5, 36, 17])
    c = Sm.correction(E, W, y)
    ref = E.astype(np.float64)[y] @ W.astype(np.float64).T      # [n][V]
    assert c.dtype == np.float32 and np.array_equal(c.astype(np.float64), ref)
    # the rank index runs over all r terms: a correction from E row y only
    E1 = np.zeros_like(E)
    E1[5] = E[5]
    assert np.array_equal(Sm.correction(E1, W, [5])[0], c[1])


def test_markov_greedy_follows_the_predecessor():
    """A correction that favours token (y_prev + 1) mod V turns greedy
    decoding of flat base logits into a cycle from the anchor."""
    V, B = 5, 7
    E = np.eye(V, dtype=np.float32)
    W = np.roll(np.eye(V, dtype=np.float32), 1, axis=0) * 3.0   # W[v, u] = 3 if v = u + 1
    z0 = np.zeros((2, B, V), dtype=np.float32)
    y, _, logq, z = Sm.sample_markov(z0, [2, 4], E, W, 0.0, 0, 0, 0)
    assert y.tolist() == [[(2 + i) % V for i in range(1, B + 1)],
                          [(4 + i) % V for i in range(1, B + 1)]]
    assert np.all(logq == 0.0)
    # top-1 support at T = 1 is the same deterministic chain
    y1, _, _, _ = Sm.sample_markov(z0, [2, 4], E, W, 1.0, 1, 9, 9)
    assert np.array_equal(y1, y)


def test_markov_joint_distribution_follows_the_factorisation():
    """Pairs (y_1, y_2) drawn over many sequences follow
    q_1(y_1) q_2(y_2 | y_1) with q_i = softmax(z_i^(0) + W_c E_c(y_{i-1})) (Eq. 8)."""
    V, r, n = 3, 2, 40_000
    g = np.random.default_rng(4)
    base = g.normal(size=(2, V)).astype(np.float32)
    E = g.normal(size=(V, r)).astype(np.float32)
    W = g.normal(size=(V, r)).astype(np.float32)
    a = 1
    y, _, logq, _ = Sm.sample_markov(np.tile(base[None], (n, 1, 1)), np.full(n, a), E, W, 1.0, 0,
                                     5, 6)
    def soft(x):
        x = x.astype(np.float64)
        p = np.exp(x - x.max())
        return p / p.sum()
    q1 = soft(base[0] + E[a] @ W.T)
    joint = np.array([[q1[u] * soft(base[1] + E[u] @ W.T)[w] for w in range(V)] for u in range(V)])
    counts = np.zeros((V, V))
    np.add.at(counts, (y[:, 0], y[:, 1]), 1)
    chi2 = scipy.stats.chisquare(counts.reshape(-1), joint.reshape(-1) * n)
    assert chi2.pvalue > 1e-3
    # log q of the second position is the log of the conditional probability
    for u in range(V):
        sel = y[:, 0] == u
        cond = soft(base[1] + E[u] @ W.T)
        assert np.allclose(logq[sel, 1], np.log(cond[y[sel, 1]]), atol=1e-5)


# ---- verification (Eq. 1-2) -------------------------------------------------------------------

def _soft(x):
    x = np.asarray(x, dtype=np.float64)
    e = np.exp(x - x.max())
    return e / e.sum()


def test_verification_preserves_the_target_distribution():
    """One candidate per round (B = 1): the first emitted token (y_1 when
    accepted, the correction token otherwise) follows p_1 exactly, whatever
    q_1 is (the property speculative sampling is built on)."""
    V, n = 5, 30_000
    g = np.random.default_rng(8)
    p_logits = g.normal(size=V).astype(np.float32)
    q_logits = g.normal(size=V).astype(np.float32)
    P = np.tile(np.stack([p_logits, g.normal(size=V).astype(np.float32)])[None], (n, 1, 1))
    Z = np.tile(q_logits[None, None], (n, 1, 1))
    y, _, _ = sample(Z.reshape(n, V), 1.0, 0, 21, 0)            # y_1 ~ q_1 per sequence
    r, tok, ratio, _ = verify(P, Z, y[:, None], 1.0, 21, 0)
    first = np.where(r == 1, y, tok)
    counts = np.bincount(first, minlength=V)
    chi2 = scipy.stats.chisquare(counts, _soft(p_logits) * n)
    assert chi2.pvalue > 1e-3
    # acceptance rate = sum_v min(p(v), q(v))
    acc = np.minimum(_soft(p_logits), _soft(q_logits)).sum()
    assert abs(r.mean() - acc) < 0.015


def test_correction_token_follows_the_residual():
    """Given a rejection, the emitted token follows [p - q]_+ normalised."""
    V, n = 4, 40_000
    p_logits = np.float32([2.0, 0.5, -1.0, 1.2])
    q_logits = np.float32([-1.0, 1.5, 0.8, 0.3])
    P = np.tile(np.stack([p_logits, p_logits])[None], (n, 1, 1))
    Z = np.tile(q_logits[None, None], (n, 1, 1))
    y = np.full((n, 1), 2)                                      # a token q likes more than p
    r, tok, _, _ = verify(P, Z, y, 1.0, 5, 1)
    rej = r == 0
    res = np.maximum(_soft(p_logits) - _soft(q_logits), 0)
    res = res / res.sum()
    counts = np.bincount(tok[rej], minlength=V)
    nz = res > 0
    assert counts[~nz].sum() == 0 and nz.sum() == 2
    chi2 = scipy.stats.chisquare(counts[nz], res[nz] * rej.sum())
    assert chi2.pvalue > 1e-3
    # rejection probability of y = 2 is 1 - p(2) / q(2)
    assert abs(rej.mean() - (1 - _soft(p_logits)[2] / _soft(q_logits)[2])) < 0.01


def test_equal_distributions_accept_everything():
    V, B, n = 6, 3, 200
    g = np.random.default_rng(9)
    Z = g.normal(size=(n, B, V)).astype(np.float32)
    P = np.concatenate([Z, g.normal(size=(n, 1, V)).astype(np.float32)], axis=1)
    y, _, _ = sample(Z.reshape(-1, V), 0.8, 0, 1, 1)
    r, tok, ratio, _ = verify(P, Z, y.reshape(n, B), 0.8, 1, 1)
    assert np.all(r == B) and np.allclose(ratio, 1.0)
    assert np.all((tok >= 0) & (tok < V))


def test_greedy_verification():
    V, B = 7, 4
    P = np.zeros((2, B + 1, V), dtype=np.float32)
    for j, v in enumerate([3, 1, 4, 1, 5]):
        P[:, j, v] = 1.0
    y = np.array([[3, 1, 4, 1], [3, 2, 4, 1]])
    r, tok, _, _ = verify(P, np.zeros((2, B, V), dtype=np.float32), y, 0.0, 0, 0)
    assert r.tolist() == [4, 1] and tok.tolist() == [5, 1]


def test_verification_noise_streams_are_their_own():
    us = {float(verify_uniform(3, 4, b, i)) for b in range(8) for i in range(1, 5)}
    assert len(us) == 32 and all(0 < u < 1 for u in us)
    g = verify_gumbel(3, 4, 0, np.arange(64))
    assert not np.array_equal(g, gumbel(3, 4, 0, np.arange(64)))


def test_bonus_token_is_the_drafting_sampler_on_the_last_row():
    """All candidates accepted: the bonus token is the plain sampler's draw
    from p_{B+1}, with the verification noise (its own counter stream)."""
    V, B = 300, 3
    g = np.random.default_rng(10)
    Z = g.normal(size=(2, B, V)).astype(np.float32)
    P = np.concatenate([Z, g.normal(size=(2, 1, V)).astype(np.float32)], axis=1)
    y, _, _ = sample(Z.reshape(-1, V), 1.0, 0, 4, 2)
    r, tok, _, _ = verify(P, Z, y.reshape(2, B), 1.0, 4, 2)
    assert np.all(r == B)
    for b in range(2):
        key = (P[b, B] / np.float32(1.0) + verify_gumbel(4, 2, b, np.arange(V))).astype(np.float32)
        assert tok[b] == int(np.argmax(key))


def test_out_of_range_candidates_are_rejected():
    V, B = 10, 2
    g = np.random.default_rng(11)
    Z = g.normal(size=(1, B, V)).astype(np.float32)
    P = np.concatenate([Z, Z[:, :1]], axis=1)
    for bad in (-1, V):
        r, tok, ratio, _ = verify(P, Z, np.array([[bad, 0]]), 1.0, 0, 0)
        assert r[0] == 0 and ratio[0, 0] == 0.0 and 0 <= tok[0] < V


def test_residual_keeps_every_positive_difference():
    """Eq. 2 is the plain positive part of p - q: a token whose target
    probability exceeds the proposal's by 2e-5 relative is the only one with
    positive residual mass, so a rejection emits it with certainty."""
    V = 6
    q_logits = np.float32([1.0, 0.5, -0.2, 0.3, 2.0, -1.0])
    P = np.tile(q_logits, (1, 2, 1)).astype(np.float32)
    P[0, 0, 1] += np.float32(2e-5)          # p(1) > q(1) by ~2e-5 relative; p < q elsewhere
    Z = q_logits[None, None].astype(np.float32)
    for seed in range(5):
        r, tok, _, _, det = verify(P, Z, np.array([[V]]), 1.0, seed, 3, detail=True)
        w = det[0]["w"]
        assert r[0] == 0 and tok[0] == 1
        assert np.count_nonzero(w) == 1 and w[1] > 0
    # with p = q exactly the residual has no mass: the bonus-rule draw from p
    P[0, 0] = q_logits
    r, tok, _, _ = verify(P, Z, np.array([[V]]), 1.0, 3, 3)
    bonus = (P[0, 0] / np.float32(1.0) + verify_gumbel(3, 3, 0, np.arange(V))).astype(np.float32)
    assert r[0] == 0 and tok[0] == int(np.argmax(bonus))


def test_residual_on_a_hand_computed_row():
    """p = (1/2, 1/4, 1/4), q = (1/4, 1/4, 1/2) from log-probabilities: the
    residual is (1/4, 0, 0), so a rejected round emits token 0; the ratio of a
    candidate 2 is p(2) / q(2) = 1/2."""
    lp = np.log(np.array([0.5, 0.25, 0.25])).astype(np.float32)
    lq = np.log(np.array([0.25, 0.25, 0.5])).astype(np.float32)
    P = np.stack([lp, lp])[None].astype(np.float32)
    Z = lq[None, None].astype(np.float32)
    seen = set()
    for seed in range(40):
        r, tok, ratio, u, det = verify(P, Z, np.array([[2]]), 1.0, seed, 0, detail=True)
        assert abs(ratio[0, 0] - 0.5) < 1e-6
        assert r[0] == (1 if u[0, 0] < ratio[0, 0] else 0)
        if r[0] == 0:
            assert tok[0] == 0
            assert np.allclose(det[0]["w"], [0.25, 0.0, 0.0], atol=1e-7)
        seen.add(int(r[0]))
    assert seen == {0, 1}


def test_top_k_proposal_is_zero_outside_the_support():
    """q over the top-k support: 0 outside it, softmax inside; a candidate
    outside the support is rejected, and the residual there equals p."""
    z = np.float32([0.3, 2.0, -1.0, 2.0, 0.9])
    q = proposal(z, 1.0, top_k=2)
    assert np.array_equal(q > 0, [False, True, False, True, False])
    assert np.allclose(q[[1, 3]], [0.5, 0.5])
    P = np.tile(np.float32([0.1, 0.2, 0.3, 0.4, 0.5]), (1, 2, 1)).astype(np.float32)
    Z = z[None, None]
    r, _, ratio, _, det = verify(P, Z, np.array([[0]]), 1.0, 1, 1, top_k=2, detail=True)
    assert r[0] == 0 and ratio[0, 0] == 0.0
    p = det[0]["p"]
    w = det[0]["w"]
    assert np.allclose(w[[0, 2, 4]], p[[0, 2, 4]]) and np.all(w[[1, 3]] == 0)


def test_top_k_verification_preserves_the_target_distribution():
    """The speculative sampling property holds for a top-k proposal too: the
    first emitted token follows p_1 exactly (chi-square), and the acceptance
    rate is sum_v min(p(v), q(v)) with q the top-k proposal."""
    V, n, k = 6, 30_000, 3
    g = np.random.default_rng(12)
    p_logits = g.normal(size=V).astype(np.float32)
    q_logits = g.normal(size=V).astype(np.float32)
    P = np.tile(np.stack([p_logits, g.normal(size=V).astype(np.float32)])[None], (n, 1, 1))
    Z = np.tile(q_logits[None, None], (n, 1, 1))
    y, _, _ = sample(Z.reshape(n, V), 1.0, k, 23, 0)            # y_1 ~ q_1 over the support
    r, tok, _, _ = verify(P, Z, y[:, None], 1.0, 23, 0, top_k=k)
    first = np.where(r == 1, y, tok)
    counts = np.bincount(first, minlength=V)
    chi2 = scipy.stats.chisquare(counts, _soft(p_logits) * n)
    assert chi2.pvalue > 1e-3
    q = np.zeros(V)
    top = np.argsort(-q_logits.astype(np.float64), kind="stable")[:k]
    q[top] = _soft(q_logits[top])
    acc = np.minimum(_soft(p_logits), q).sum()
    assert abs(r.mean() - acc) < 0.015
