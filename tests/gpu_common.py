"""Helpers of the GPU parity tests: drive the HIP views and the oracle views
with the same seeded inputs (drawn once, on the GPU, and copied to the host
for the oracle), and compare logits per row against the tolerances of the
drafting step."""
from __future__ import annotations

import numpy as np
import torch

import synth
from oracle import sample as OS
from oracle import views as OV


class Pair:
    """GPU views of `batch` sequences plus the oracle's views of the same rows."""

    def __init__(self, ldr, shape, batch, G, oracle_seqs=None):
        self.ldr, self.s, self.batch = ldr, shape, batch
        self.G = G
        self.G64 = None if G is None else synth.to_f64(G)
        self.views = ldr.Views(shape, batch, G).init()
        self.seqs = list(range(batch)) if oracle_seqs is None else list(oracle_seqs)
        self.ost = {b: OV.empty(shape) for b in self.seqs}

    def ingest(self, n, K, V, h):
        """n: list of per-sequence row counts (<= K.shape[1])."""
        nt = torch.tensor(n, dtype=torch.int32, device=K.device)
        self.views.update(nt, K, V, h)
        for b in self.seqs:
            nb = int(n[b])
            self.ost[b] = OV.update(self.s, self.ost[b], self.G64, synth.to_f64(K[b, :nb]),
                                    synth.to_f64(V[b, :nb]),
                                    synth.to_f64(h[b]) if nb > 0 else self.ost[b].h)

    def prefill(self, prefix, chunk, ragged=0):
        """Ingest a synthetic prefix in chunks; sequence b gets `ragged * b` fewer rows
        in the last chunk."""
        for i, (K, V, h) in enumerate(synth.prefix_chunks(self.s, self.batch, prefix, chunk,
                                                          device="cuda")):
            n = [K.shape[1]] * self.batch
            if ragged and (i + 1) * chunk >= prefix:
                n = [max(0, K.shape[1] - ragged * b) for b in range(self.batch)]
            self.ingest(n, K, V, h)

    def decode(self, steps, n_max, rng):
        for st in range(steps):
            K, V, h = synth.decode_rows(self.s, self.batch, n_max, st, device="cuda")
            n = [int(x) for x in rng.integers(0, n_max + 1, self.batch)]
            self.ingest(n, K, V, h)


def check_views(pair, rtol_m=1e-4, atol_m=1e-6):
    """Positions, window and boundary bit-exact, summary within tolerance; a
    view the shape drops (ablation variants) has no region to compare."""
    torch.cuda.synchronize()
    v = pair.views
    pos = v.pos.cpu().numpy()
    win, summ, bnd, pool = v.window(), v.summary(), v.boundary(), v.pooled()
    PK, PV = (t.cpu() for t in pool) if pool is not None else (None, None)
    bf16 = pair.s.dtype == "bf16"
    Kw, Vw = (t.cpu() for t in win) if win is not None else (None, None)
    M, eta = (t.cpu().numpy() for t in summ) if summ is not None else (None, None)
    hb = bnd.cpu() if bnd is not None else None
    for b in pair.seqs:
        o = pair.ost[b]
        assert pos[b] == o.t, (b, pos[b], o.t)
        # window rows and boundary states are copies: bit-exact
        if Kw is not None:
            assert np.array_equal(synth.to_f64(Kw[b]), o.Kw), f"window K of sequence {b}"
            assert np.array_equal(synth.to_f64(Vw[b]), o.Vw), f"window V of sequence {b}"
        if hb is not None:
            assert np.array_equal(synth.to_f64(hb[b]), o.h), f"boundary of sequence {b}"
        if PK is not None:
            # slot means: fp32 sums and one division, stored in the model dtype
            rtol = 2.0 ** -8 if bf16 else 1e-6
            np.testing.assert_allclose(synth.to_f64(PK[b]), o.PK, rtol=rtol, atol=2e-5)
            np.testing.assert_allclose(synth.to_f64(PV[b]), o.PV, rtol=rtol, atol=2e-5)
        if M is None:
            continue
        if o.t == 0:
            assert np.all(np.isneginf(eta[b]))
            assert np.all(M[b] == 0)
            continue
        np.testing.assert_allclose(eta[b], o.eta, rtol=1e-5, atol=1e-5)
        scale = np.abs(o.M).max()
        np.testing.assert_allclose(M[b], o.M, rtol=rtol_m, atol=atol_m * max(scale, 1.0))


def row_errors(z_gpu, z_ref):
    """Per row: max |dz| / max |z_ref| and the cosine similarity."""
    z_gpu = np.asarray(z_gpu, dtype=np.float64)
    z_ref = np.asarray(z_ref, dtype=np.float64)
    err = np.abs(z_gpu - z_ref).max(axis=-1) / np.abs(z_ref).max(axis=-1)
    cos = (z_gpu * z_ref).sum(-1) / (np.linalg.norm(z_gpu, axis=-1) *
                                     np.linalg.norm(z_ref, axis=-1))
    return err, cos


def check_logits(z_gpu, z_ref, shape):
    err, cos = row_errors(z_gpu, z_ref)
    if shape.dtype == "f32":
        assert err.max() <= 1e-4, err.max()
    else:
        assert err.max() <= 2e-2, err.max()
        assert cos.min() >= 0.999, cos.min()
    return err, cos


class LazyRows:
    """Rows of a device tensor converted to float64 on indexing."""

    def __init__(self, t):
        self.t = t

    def __getitem__(self, idx):
        if isinstance(idx, np.ndarray):
            idx = torch.from_numpy(idx).to(self.t.device)
        return synth.to_f64(self.t[idx])


class LazyLayers:
    def __init__(self, layers):
        self.layers = layers

    def __getitem__(self, j):
        return {k: synth.to_f64(v) for k, v in self.layers[j].items()}

    def __len__(self):
        return len(self.layers)


def lazy_weights_f64(w):
    """A weight dict for the oracle whose big tensors are converted on access."""
    out = {k: synth.to_f64(v) for k, v in w.items()
           if k not in ("layers", "embed", "lm_head")}
    out["embed"] = LazyRows(w["embed"])
    out["lm_head"] = LazyRows(w["lm_head"])
    out["layers"] = LazyLayers(w["layers"])
    return out


def residual_decision(d, bonus_tok, rel_err, key_abs=1e-5):
    """(clean, valid tokens) of a residual draw (Eq. 2) from the oracle's
    float64 stop row d = {p, q, w, g}, when the kernel's p_v and q_v are each
    within rel_err (relative) of the oracle's: token v's key log w_v + g_v
    then lies in [log(w_v - e_v), log(w_v + e_v)] + g_v, e_v = rel_err
    max(p_v, q_v). Clean: the oracle's token has a lower bound above every
    other token's upper bound and some w_v exceeds e_v (so the kernel's
    residual cannot be empty); the kernel must then emit the oracle's token.
    Otherwise the valid tokens are those whose upper bound reaches the best
    lower bound, plus the bonus-rule draw when every w_v is within e_v."""
    p, q, w, g = d["p"], d["q"], d["w"], d["g"]
    e = rel_err * np.maximum(p, q)
    with np.errstate(divide="ignore"):
        lo = np.where(w > e, np.log(np.maximum(w - e, 1e-300)), -np.inf) + g - key_abs
        hi = np.where(w + e > 0, np.log(w + e), -np.inf) + g + key_abs
    can_be_empty = not np.any(w > e)
    best_lo = lo.max()
    valid = set(np.flatnonzero(hi >= best_lo).tolist()) if np.isfinite(best_lo) else \
        set(np.flatnonzero(np.isfinite(hi)).tolist())
    if can_be_empty:
        valid.add(int(bonus_tok))
    t = int(np.argmax(lo))
    clean = (not can_be_empty) and lo[t] > np.max(np.delete(hi, t))
    return clean, valid


# fp32 slack of a GPU chunk key: its log-mass is an fp32 sum of 16 exponentials
# and an fp32 logarithm (a few ulp of |L|, |L| up to ~30 here)
CHUNK_KEY_ABS, CHUNK_KEY_REL = 2e-5, 2e-6


def draw_near_tie(z_ref, y_ref, y_gpu, row, T, seed, step, e, top_k=0):
    """Asserts that the GPU token y_gpu, drawn with the oracle's noise from
    logits within e (max |dz| / T) of the oracle's z_ref [V], is the oracle's
    two-level draw y_ref or a near tie of it at the level where the two part:
    the chunk keys L_c + h_c of the two chunks within 2e plus the fp32 slack of
    a chunk key (a log-mass moves by at most max |dz| / T), then the token keys
    z_v / T + g_v inside the GPU's chunk within 2e of that chunk's best.
    Returns True where the tokens differ."""
    if y_gpu == y_ref:
        return False
    z = np.asarray(z_ref, dtype=np.float64)
    V = z.shape[0]
    inside = np.zeros((1, V), dtype=bool)
    inside[0, OS.support(np.asarray(z_ref, dtype=np.float32), top_k)] = True
    T32 = float(np.float32(T))
    assert inside[0, y_gpu], (row, y_gpu)
    c_o, c_g = int(y_ref) // OS.CHUNK, int(y_gpu) // OS.CHUNK
    if c_o != c_g:
        L = OS.chunk_log_mass(z[None] / T32, inside)[0]
        h = OS.gumbel(seed, step, row, np.array([c_o, c_g]), stream=OS.CHUNK_STREAM)
        k = L[[c_o, c_g]] + h.astype(np.float64)
        slack = CHUNK_KEY_ABS + CHUNK_KEY_REL * np.abs(k).max()
        assert k[0] - k[1] <= 2 * e + slack, (row, c_o, c_g, k[0] - k[1], e)
    v = np.arange(c_g * OS.CHUNK, min(V, (c_g + 1) * OS.CHUNK))
    v = v[inside[0, v]]
    key = z[v] / T32 + OS.gumbel(seed, step, row, v).astype(np.float64)
    kg = key[list(v).index(int(y_gpu))]
    assert key.max() - kg <= 2 * e + 1e-6, (row, int(v[np.argmax(key)]), int(y_gpu), e)
    return True
