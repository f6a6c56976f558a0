"""Oracle for per-position sampling of the factorised proposal (Eq. 8).

This file is test infrastructure: only the tests, the smoke check and the
benchmark's CPU baseline use it; the library never does.

Each drafted position i of each sequence is one row of base logits z
(fp32, [V]). For temperature T > 0 the proposal is q_i = softmax(z/T) over a
support S (all V tokens, or the top_k largest logits, lower index first on
ties). The paper fixes only q_i; the draw is a two-level Gumbel-max, which is
an exact sample of q_i:

* the vocabulary is cut into chunks of C = 16 consecutive tokens
  (chunk c = tokens 16c .. 16c + 15, the last one ragged);
* each chunk's log-mass L_c = log sum_{v in c, v in S} exp(z_v/T) (-inf for
  a chunk with no support token);
* the chunk c* = argmax_c (L_c + h_c), h_c standard Gumbel noise: the maximum
  of independent Gumbels shifted by L_c picks c with probability
  exp(L_c) / sum exp(L), i.e. q_i(c);
* the token y = argmax_{v in c*, v in S} (z_v/T + g_v), g_v Gumbel noise
  independent of h: y given c* has probability exp(z_y/T - L_c*), so
  P(y) = q_i(y).

T = 0 is greedy: y = argmax_v z_v (lowest index on ties), q a point mass. The
row also yields lse = log sum_{v in S} exp(z_v/T) and log q(y) = z_y/T - lse,
which the verifier's acceptance test and residual (Eq. 1-2) need.

Both argmaxes are integer decisions taken from fp32 keys, so the keys are
fp32 as the GPU kernel computes them: the token keys fl(fl(z_v / T) + g_v),
every step an IEEE fp32 operation, and the chunk keys fl(fl32(L_c) + h_c)
with L_c computed here in float64 and rounded to fp32 (the kernel sums the
chunk's 16 exponentials in fp32, so its L_c can differ in the last bits: its
chunk choice can differ from this one only where two chunk keys tie within
that error). Ties go to the lower index at both levels. The noise is fully
specified here:

* bits: Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers:
  as easy as 1, 2, 3", SC 2011) with key (seed mod 2^32, seed div 2^32) and
  counter (v div 4, row, step mod 2^32, (step div 2^32) mod 2^30 + 2^30 s),
  s the stream; entry v takes output word v mod 4. Token noise g_v is entry
  v of stream 0, chunk noise h_c entry c of stream 3;
* uniform: k = bits >> 9, u = (2k + 1) * 2^-24, exact in fp32, in (0, 1);
* Gumbel: -log(-log(u)) with the fp32 logarithm ``logf`` below, a fixed
  sequence of IEEE fp32 operations (no fused multiply-add): exponent split,
  mantissa folded into [sqrt(1/2), sqrt(2)], then 2 atanh(f), f = (m-1)/(m+1),
  by its odd power series to the f^11 term.

lse and log q are computed in float64 here.

Markov-corrected sampling (Eq. 7-8): with y_0 the anchor, position i's logits
are z_i = z_i^(0) + W_c E_c(y_{i-1}) and y_i is drawn from softmax(z_i / T)
as above, so positions are taken in order. The correction c = W_c E_c(y) is,
for each vocabulary entry v, the sum over the rank index k = 0, 1, ..., r-1
in that order of the fp32 products W_c[v, k] E_c[y, k], every product and
partial sum rounded to fp32 (none fused), and z_i = fl(z_i^(0) + c): the
corrected logits, like the keys, are a fixed sequence of IEEE fp32 operations.
Position i of sequence b uses the noise row b B + i - 1, the plain sampler's
row of that logit row.
"""
from __future__ import annotations

import numpy as np
import scipy.special

# Philox4x32 multipliers and Weyl key increments (Salmon et al., SC 2011).
PHILOX_M0 = np.uint64(0xD2511F53)
PHILOX_M1 = np.uint64(0xCD9E8D57)
PHILOX_W0 = np.uint64(0x9E3779B9)
PHILOX_W1 = np.uint64(0xBB67AE85)
_M32 = np.uint64(0xFFFFFFFF)
_S32 = np.uint64(32)


def philox4x32_10(ctr, key):
    """Philox4x32 with 10 rounds. ctr: 4 arrays of 32-bit words, key: 2 (held
    in uint64, broadcastable). Returns the 4 output words (uint64 < 2^32).
    A round: (hi0, lo0) = M0 c0, (hi1, lo1) = M1 c2 (64-bit products, exact in
    uint64), c <- (hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0); the key advances by
    the Weyl constants before every round but the first."""
    c = [np.asarray(x, dtype=np.uint64) & _M32 for x in ctr]
    k0, k1 = (np.asarray(x, dtype=np.uint64) & _M32 for x in key)
    for rnd in range(10):
        if rnd:
            k0 = (k0 + PHILOX_W0) & _M32
            k1 = (k1 + PHILOX_W1) & _M32
        p0 = c[0] * PHILOX_M0
        p1 = c[2] * PHILOX_M1
        c = [(p1 >> _S32) ^ c[1] ^ k0, p1 & _M32, (p0 >> _S32) ^ c[3] ^ k1, p0 & _M32]
    return c


def _counter(seed, step, stream):
    """Key and the two upper counter words of a (seed, step, stream)."""
    seed, step = int(seed), int(step)
    key = (np.uint64(seed & 0xFFFFFFFF), np.uint64((seed >> 32) & 0xFFFFFFFF))
    c2 = np.uint64(step & 0xFFFFFFFF)
    c3 = np.uint64(((step >> 32) & 0x3FFFFFFF) | (int(stream) << 30))
    return key, c2, c3


# fp32 constants of logf, as bit patterns (nearest fp32 to the exact value).
def _f(bits):
    return np.array(bits, dtype=np.uint32).view(np.float32)[()]


C3, C5, C7, C9, C11 = (_f(0x3EAAAAAB), _f(0x3E4CCCCD), _f(0x3E124925), _f(0x3DE38E39),
                       _f(0x3DBA2E8C))                          # 1/3, 1/5, 1/7, 1/9, 1/11
LN2_HI = _f(0x3F317200)    # ln 2 to 16 bits: e * LN2_HI is exact for |e| <= 255
LN2_LO = _f(0x35BFBE8E)    # ln 2 - LN2_HI
SQRT2 = _f(0x3FB504F3)
ONE, TWO, HALF = np.float32(1.0), np.float32(2.0), np.float32(0.5)


def logf(x):
    """Natural log of positive normal fp32 values, as a fixed sequence of
    IEEE fp32 operations (each rounded to nearest, none fused).

    x = 2^e * m, m in [1, 2); if m > sqrt(2): m /= 2, e += 1. Then
    log x = e ln2 + 2 atanh(f), f = (m - 1) / (m + 1), |f| <= 0.1716, and
    2 atanh(f) = 2f (1 + s/3 + s^2/5 + s^3/7 + s^4/9 + s^5/11), s = f^2
    (truncation below 1e-10 relative)."""
    x = np.asarray(x, dtype=np.float32)
    bits = x.view(np.uint32)
    e = (((bits >> np.uint32(23)) & np.uint32(0xFF)).astype(np.int32) - 127)
    m = ((bits & np.uint32(0x7FFFFF)) | np.uint32(0x3F800000)).view(np.float32)
    big = m > SQRT2
    m = np.where(big, m * HALF, m)
    e = (e + big.astype(np.int32)).astype(np.float32)
    f = (m - ONE) / (m + ONE)
    s = f * f
    p = C11
    p = p * s + C9
    p = p * s + C7
    p = p * s + C5
    p = p * s + C3
    p = p * s + ONE
    r = (f * TWO) * p
    return (e * LN2_HI + (e * LN2_LO + r)).astype(np.float32)


def philox_bits(seed, step, row, v, stream=0):
    """The 32 noise bits of token v in row `row` of a stream (uint32 arrays)."""
    v, row = np.broadcast_arrays(np.asarray(v, dtype=np.uint64),
                                 np.asarray(row, dtype=np.uint64))
    key, c2, c3 = _counter(seed, step, stream)
    w = np.stack(philox4x32_10((v >> np.uint64(2), row, c2 + 0 * v, c3 + 0 * v), key), axis=0)
    word = np.take_along_axis(w, (v & np.uint64(3)).astype(np.int64)[None], axis=0)[0]
    return word.astype(np.uint32)


def uniform(bits):
    """u = (2 (bits >> 9) + 1) 2^-24, exact in fp32, strictly inside (0, 1)."""
    k = (np.asarray(bits, dtype=np.uint32) >> np.uint32(9)).astype(np.float32)
    return ((k * TWO + ONE) * np.float32(2.0 ** -24)).astype(np.float32)


def gumbel(seed, step, row, v, stream=0):
    """-log(-log(u)) in fp32 for entry (entries) v of row `row` of a stream:
    stream 0 holds the token noise g_v, stream 3 the chunk noise h_c."""
    u = uniform(philox_bits(seed, step, row, v, stream))
    return -logf(-logf(u))


CHUNK = 16          # tokens per vocabulary chunk of the two-level draw
CHUNK_STREAM = 3    # noise stream of the chunk keys


def support(z, top_k):
    """Token ids in the support: all, or the top_k largest z (lower index
    first among equal values)."""
    V = z.shape[0]
    if top_k <= 0 or top_k >= V:
        return np.arange(V)
    return np.sort(np.argsort(-z.astype(np.float64), kind="stable")[:top_k])


def chunk_log_mass(zt, inside, chunk=CHUNK):
    """L_c = log sum over the support tokens of chunk c of exp(zt_v), float64
    [n][ceil(V / chunk)], -inf for a chunk without support tokens. zt: [n][V]
    scaled logits, inside: [n][V] support mask."""
    n, V = zt.shape
    nch = -(-V // chunk)
    x = np.full((n, nch * chunk), -np.inf)
    x[:, :V] = np.where(inside, np.asarray(zt, dtype=np.float64), -np.inf)
    with np.errstate(divide="ignore"):
        return scipy.special.logsumexp(x.reshape(n, nch, chunk), axis=2)


def chunk_keys(L, seed, step, rows):
    """fp32 chunk keys fl(fl32(L_c) + h_c) of [n][nch] log-masses for the
    noise rows `rows`; -inf where L_c = -inf."""
    n, nch = L.shape
    h = gumbel(seed, step, np.asarray(rows)[:, None], np.arange(nch)[None, :], CHUNK_STREAM)
    with np.errstate(invalid="ignore"):
        return (np.asarray(L, dtype=np.float32) + h).astype(np.float32)


def draw_in_chunks(zt, inside, c, seed, step, rows, chunk=CHUNK):
    """The token of chunk c[i] of each row i: first argmax of the fp32 keys
    fl(zt_v + g_v) over the chunk's support tokens."""
    n, V = zt.shape
    v = np.asarray(c)[:, None] * chunk + np.arange(chunk)[None, :]
    valid = v < V
    v = np.minimum(v, V - 1)
    key = (np.take_along_axis(zt, v, 1) +
           gumbel(seed, step, np.asarray(rows)[:, None], v)).astype(np.float32)
    key = np.where(valid & np.take_along_axis(inside, v, 1), key, -np.inf)
    return v[np.arange(n), np.argmax(key, axis=1)]


def sample(logits, temperature, top_k, seed, step, rows=None, chunk=CHUNK, rows_per_pass=16,
           detail=False):
    """Tokens (int64), lse and log q (float64) for the rows of a [n][V] fp32
    logits array, drawn by the two-level Gumbel-max over chunks of `chunk`
    tokens. `rows` gives each row's index in the noise counter (default
    0..n-1). detail=True appends, for T > 0, the fp32 chunk keys [n][nch]
    and the chosen chunks [n]."""
    z = np.asarray(logits, dtype=np.float32)
    n, V = z.shape
    rows = np.arange(n) if rows is None else np.asarray(rows)
    if temperature == 0.0:
        y = np.argmax(z, axis=1)                                # first maximum
        out = (y.astype(np.int64), z[np.arange(n), y].astype(np.float64), np.zeros(n))
        return out + (None, None) if detail else out
    T = np.float32(temperature)
    ys, lses, keys, cs = [], [], [], []
    for a in range(0, n, rows_per_pass):
        zc = z[a:a + rows_per_pass]
        zt = (zc / T).astype(np.float32)                       # IEEE fp32 division
        inside = np.zeros(zc.shape, dtype=bool)
        for i in range(zc.shape[0]):
            inside[i, support(zc[i], top_k)] = True
        K = chunk_keys(chunk_log_mass(zt, inside, chunk), seed, step, rows[a:a + rows_per_pass])
        c = np.argmax(K, axis=1)                               # first maximum
        ys.append(draw_in_chunks(zt, inside, c, seed, step, rows[a:a + rows_per_pass], chunk))
        zs = np.where(inside, zc.astype(np.float64) / float(T), -np.inf)
        lses.append(scipy.special.logsumexp(zs, axis=1))
        keys.append(K)
        cs.append(c)
    y = np.concatenate(ys).astype(np.int64)
    lse = np.concatenate(lses)
    out = (y, lse, z[np.arange(n), y].astype(np.float64) / float(T) - lse)
    if detail:
        out = out + (np.concatenate(keys), np.concatenate(cs).astype(np.int64))
    return out


def sample_row(z, temperature, top_k, seed, step, row):
    """(token, lse, logq) for one row of fp32 logits z [V]."""
    y, lse, logq = sample(np.asarray(z, dtype=np.float32)[None], temperature, top_k, seed,
                          step, rows=[row])
    return int(y[0]), float(lse[0]), float(logq[0])


def correction(E_c, W_c, y):
    """c = W_c E_c(y) (Eq. 7) for the previous tokens y [n]: fp32 [n][V], each
    entry summed over the rank index in order, products and sums in fp32."""
    E = np.asarray(E_c, dtype=np.float32)          # [V][r]
    W = np.asarray(W_c, dtype=np.float32)          # [V][r]
    e = E[np.asarray(y, dtype=np.int64)]           # [n][r]
    c = np.zeros((e.shape[0], W.shape[0]), dtype=np.float32)
    for k in range(W.shape[1]):
        c = (c + (W[None, :, k] * e[:, k, None]).astype(np.float32)).astype(np.float32)
    return c


def sample_markov(z0, anchor, E_c, W_c, temperature, top_k, seed, step):
    """Sequential sampling of the corrected proposal (Eq. 7-8) for base logits
    z0 [batch][B][V] (fp32) and anchors [batch]. Returns tokens [batch][B]
    (int64), lse and log q [batch][B] (float64) of the corrected rows, and the
    corrected logits [batch][B][V] (fp32)."""
    z0 = np.asarray(z0, dtype=np.float32)
    nb, B, V = z0.shape
    y_prev = np.asarray(anchor, dtype=np.int64)
    toks = np.zeros((nb, B), dtype=np.int64)
    lses = np.zeros((nb, B))
    logqs = np.zeros((nb, B))
    z = np.empty_like(z0)
    for i in range(B):
        zi = (z0[:, i, :] + correction(E_c, W_c, y_prev)).astype(np.float32)
        y, lse, logq = sample(zi, temperature, top_k, seed, step, rows=np.arange(nb) * B + i)
        toks[:, i], lses[:, i], logqs[:, i], z[:, i, :] = y, lse, logq, zi
        y_prev = y
    return toks, lses, logqs, z


# ---- verification (Eq. 1-2) -------------------------------------------------------------------
#
# The target scores [a, y_1 .. y_B] in one pass and gives B + 1 distributions:
# row j of the target logits P is p_{j+1}. Candidate y_i is accepted when
# u_i < p_i(y_i) / q_i(y_i) (Eq. 1), tested in order; at the first rejection
# the round emits a token drawn from the residual w = [p_i - q_i]_+ normalised
# (Eq. 2), and after B acceptances a bonus token drawn from p_{B+1}. p and q
# take the same temperature T: p_i = softmax(P_i / T) over the whole
# vocabulary, q_i = softmax(z_i / T) over the drafting sampler's support S_i
# (all tokens, or the top_k largest z_i, lower index first on ties) and 0
# outside it. The ratio, p, q and the residual are float64 here; the residual
# is the plain positive part of p - q, with no threshold.
#
# Readings where the paper is silent:
#  * a candidate outside [0, V), or outside the support S_i, has q = 0 (the
#    proposal cannot produce it) and is rejected;
#  * a residual with no positive entry (p_i = q_i exactly, where a rejection
#    has probability zero) draws from p_i with the bonus rule instead;
#  * the bonus token is drawn by a one-level Gumbel-max over the whole
#    vocabulary, from the fp32 keys fl(fl(P_v / T) + g_v), first maximum; the
#    correction token is the first maximum of log w_v + g_v over the tokens
#    with w_v > 0;
#  * T = 0 verifies greedily: y_i is accepted when it is the first argmax of
#    P_i, and the round emits the first argmax of the row where it stops.
#
# Noise (the drafting layout of Philox4x32-10 in streams of its own):
#  * u_i of sequence b: word 0 of the block of counter i - 1 and row b in
#    stream 1, made uniform like the drafting noise;
#  * the emitted token's Gumbel noise g_v: token v of row b in stream 2.


def verify_uniform(seed, step, b, i):
    """u_i of sequence b (i = 1 .. B) as an exact fp32 value in (0, 1)."""
    key, c2, c3 = _counter(seed, step, 1)
    w = philox4x32_10((np.uint64(i - 1), np.uint64(b), c2, c3), key)
    return uniform(np.uint32(int(w[0])))


def verify_gumbel(seed, step, b, v):
    """Gumbel noise of token(s) v for the emitted token of sequence b."""
    return -logf(-logf(uniform(philox_bits(seed, step, b, v, stream=2))))


def _softmax64(x):
    x = np.asarray(x, dtype=np.float64)
    m = x.max()
    e = np.exp(x - m)
    return e / e.sum()


def proposal(z, temperature, top_k=0):
    """q = softmax(z / T) over the support of z (top_k as in ``support``),
    0 outside it: float64 [V]."""
    z = np.asarray(z, dtype=np.float32)
    q = np.zeros(z.shape[0])
    s = support(z, top_k)
    q[s] = _softmax64(z[s].astype(np.float64) / float(np.float32(temperature)))
    return q


def verify(P, Z, y, temperature, seed, step, keys=False, top_k=0, detail=False):
    """Speculative verification of one round for every sequence.
    P: target logits [batch][B + 1][V]; Z: draft logits [batch][B][V] (the
    proposal q_i = softmax(z_i / T) over the top_k support, see ``proposal``);
    y: drafted tokens [batch][B].
    Returns (r [batch] accepted counts, token [batch] emitted after them,
    ratio [batch][B] p_i(y_i) / q_i(y_i) in float64, u [batch][B]); ratio and
    u are 0 past the first rejection and at T = 0. keys=True appends the list
    of each sequence's keys over the row it emits from (float64 [V]; the
    token is their first argmax). detail=True appends, per sequence, a dict
    with the stop row's p, q, residual w (None after B acceptances) and the
    emission noise g."""
    P = np.asarray(P, dtype=np.float32)
    Z = np.asarray(Z, dtype=np.float32)
    y = np.asarray(y, dtype=np.int64)
    nb, B1, V = P.shape
    B = B1 - 1
    r = np.zeros(nb, dtype=np.int64)
    tok = np.zeros(nb, dtype=np.int64)
    ratio = np.zeros((nb, B))
    us = np.zeros((nb, B))
    all_keys, details = [], []
    for b in range(nb):
        if temperature == 0.0:
            i = 0
            while i < B and int(np.argmax(P[b, i])) == y[b, i]:
                i += 1
            r[b], tok[b] = i, int(np.argmax(P[b, i]))
            all_keys.append(P[b, i].astype(np.float64))
            details.append(None)
            continue
        T = np.float32(temperature)
        stop = B
        for i in range(B):
            p = _softmax64(P[b, i].astype(np.float64) / float(T))
            q = proposal(Z[b, i], T, top_k)
            yi = int(y[b, i])
            ratio[b, i] = p[yi] / q[yi] if 0 <= yi < V and q[yi] > 0 else 0.0
            us[b, i] = float(verify_uniform(seed, step, b, i + 1))
            if not us[b, i] < ratio[b, i]:
                stop = i
                break
        r[b] = stop
        g = verify_gumbel(seed, step, b, np.arange(V))
        w = p = q = None
        if stop < B:
            p = _softmax64(P[b, stop].astype(np.float64) / float(T))
            q = proposal(Z[b, stop], T, top_k)
            w = np.maximum(p - q, 0.0)                           # Eq. 2: [p - q]_+
        if w is not None and np.any(w > 0):
            key = np.full(V, -np.inf)
            key[w > 0] = np.log(w[w > 0]) + g[w > 0].astype(np.float64)
        else:
            key = P[b, stop] / T + g                               # fp32, as the sampler
        tok[b] = int(np.argmax(key))
        all_keys.append(key.astype(np.float64))
        details.append({"p": p, "q": q, "w": w, "g": g.astype(np.float64)})
    out = (r, tok, ratio, us)
    if keys:
        out = out + (all_keys,)
    if detail:
        out = out + (details,)
    return out
