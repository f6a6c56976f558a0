"""GPU parity of speculative verification (Eq. 1-2) against the oracle, fed
the same seeded fp32 logits and candidates.

The oracle takes every decision in float64 from Eq. 1-2 as written; the
kernels take them from fp32 values. Counts and tokens must agree exactly
wherever the decision has a margin above the fp32 error:

* acceptance: the ratio p_i(y_i) / q_i(y_i) more than RATIO_TOL (relative)
  away from u_i;
* residual draw: the GPU's residual entries w_v = p_v - q_v are fp32
  differences of two fp32 probabilities, each within REL_ERR of the exact
  value (the normalisers are fp32 sums over the vocabulary), so token v's key
  log w_v + g_v lies in [log(w_v - e_v), log(w_v + e_v)] + g_v with
  e_v = REL_ERR max(p_v, q_v) (an entry with w_v <= e_v may be positive or not
  on the GPU). The draw is clean when the oracle's token has a lower bound
  above every other token's upper bound and some entry has w_v > e_v (so the
  GPU cannot see an empty residual); then the tokens must be equal. Otherwise
  (a near tie) the GPU token must be one whose upper bound reaches the best
  lower bound, or the bonus-rule draw when every entry is within e_v;
* bonus draws: the keys are the same fp32 operations on both sides, so the
  tokens agree exactly.

n_new is always r + 1."""
import numpy as np
import pytest
import torch

import synth
from gpu_common import residual_decision
from oracle import sample as OS

pytestmark = pytest.mark.gpu

RATIO_TOL = 1e-4
REL_ERR = 2e-5       # relative error bound of the kernels' fp32 p_v and q_v
KEY_ABS = 1e-5       # rounding of the fp32 key log(w) + g


def _run(ldr, y, z, P, T, seed, step, top_k=0):
    batch, B, V = z.shape
    lse = None
    if T > 0:
        lse = ldr.sample(z.reshape(-1, V), T, top_k, seed=seed + 1, step=step)[1].reshape(batch, B)
    acc, tok, n_new = ldr.verify(P, z if T > 0 else None, lse, y, T, seed, step, top_k=top_k)
    torch.cuda.synchronize()
    return acc.cpu().numpy(), tok.cpu().numpy(), n_new.cpu().numpy()


def _residual_decision(d, bonus_tok):
    return residual_decision(d, bonus_tok, REL_ERR, KEY_ABS)


def _compare(acc, tok, n_new, y, z, P, T, seed, step, max_ties=1, top_k=0):
    """Counts and tokens against the oracle; returns (oracle r, oracle token,
    indices of the sequences decided without a near tie)."""
    Pn, zn = P.cpu().numpy(), z.cpu().numpy()
    r, t, ratio, u, keys, det = OS.verify(Pn, zn, y.cpu().numpy(), T, seed, step, keys=True,
                                          top_k=top_k, detail=True)
    B = z.shape[1]
    V = z.shape[2]
    assert np.array_equal(n_new, acc + 1)
    assert np.all((acc >= 0) & (acc <= B))
    ties, clean = 0, []
    for b in range(len(r)):
        n = min(r[b] + 1, B)                    # decisions taken up to the stop
        margin = np.abs(ratio[b, :n] - u[b, :n]) / np.maximum(1.0, ratio[b, :n])
        if T > 0 and np.any(margin <= RATIO_TOL):
            ties += 1
            continue
        assert acc[b] == r[b], (b, acc[b], r[b])
        if T == 0 or r[b] == B:                 # argmax / bonus keys: the same fp32 values
            assert tok[b] == t[b], (b, tok[b], t[b])
            clean.append(b)
            continue
        g = OS.verify_gumbel(seed, step, b, np.arange(V))
        bonus_tok = int(np.argmax(Pn[b, r[b]] / np.float32(T) + g))
        is_clean, valid = _residual_decision(det[b], bonus_tok)
        if is_clean:
            assert tok[b] == t[b], (b, tok[b], t[b])
            clean.append(b)
        else:
            ties += 1
            assert int(tok[b]) in valid, (b, tok[b], t[b])
    assert ties <= max_ties, ties
    return r, t, clean


@pytest.mark.parametrize("batch,B,V,T", [(3, 4, 1003, 1.0), (5, 7, 4096, 0.7), (2, 1, 257, 1.0),
                                         (9, 16, 2000, 1.3), (1, 70, 515, 1.0)])
def test_verify_matches_oracle(gpu_lib, batch, B, V, T):
    y, z, P = synth.verify_round(batch, B, V, seed=batch * 31 + B + V, device="cuda")
    for step in range(3):
        acc, tok, n_new = _run(gpu_lib, y, z, P, T, seed=11, step=step)
        _compare(acc, tok, n_new, y, z, P, T, 11, step)


def test_verify_full_size(gpu_lib):
    """Qwen3 vocabulary, batch 16, block 16: every count and token."""
    y, z, P = synth.verify_round(16, 16, 151936, device="cuda")
    acc, tok, n_new = _run(gpu_lib, y, z, P, 1.0, seed=5, step=2)
    r, _, _ = _compare(acc, tok, n_new, y, z, P, 1.0, 5, 2)
    assert len(set(r.tolist())) > 3          # the round lengths vary


@pytest.mark.parametrize("batch,B,V", [(4, 5, 999), (3, 16, 151936), (2, 80, 300)])
def test_greedy_verify(gpu_lib, batch, B, V):
    y, z, P = synth.verify_round(batch, B, V, seed=7 + B, device="cuda")
    # candidates equal to the target's argmax up to a sequence-dependent length
    am = P[:, :B].argmax(dim=2).to(torch.int32)
    for b in range(batch):
        cut = (b * 3) % (B + 1)
        y[b, :cut] = am[b, :cut]
    P[0, 0, 5] = P[0, 0].max()                # a tie: the lower index is the argmax
    acc, tok, n_new = _run(gpu_lib, y, z, P, 0.0, seed=0, step=0)
    r, t, _, _ = OS.verify(P.cpu().numpy(), z.cpu().numpy(), y.cpu().numpy(), 0.0, 0, 0)
    assert np.array_equal(acc, r) and np.array_equal(tok, t) and np.array_equal(n_new, r + 1)


def test_equal_distributions_accept_all_and_draw_the_bonus(gpu_lib):
    batch, B, V = 6, 8, 4096
    y, z, P = synth.verify_round(batch, B, V, seed=3, device="cuda")
    P[:, :B] = z
    acc, tok, n_new = _run(gpu_lib, y, z, P, 1.0, seed=9, step=4)
    r, t, clean = _compare(acc, tok, n_new, y, z, P, 1.0, 9, 4)
    assert np.all(r == B) and len(clean) >= batch - 1
    assert np.all(acc[clean] == B)


def test_out_of_range_candidates_and_empty_residual(gpu_lib):
    """Rows where p = q exactly in fp32 and float64 (three tokens at logit 0,
    the rest far below, so both normalisers are log 3 exactly on both sides):
    a forced rejection leaves a residual with no positive entry, and the
    round draws from p by the bonus rule, bit-exact."""
    batch, B, V = 3, 4, 1000
    y, z, P = synth.verify_round(batch, B, V, seed=4, device="cuda")
    z.fill_(-1e4)
    z[:, :, 7] = 0.0
    z[:, :, 100] = 0.0
    z[:, :, 901] = 0.0
    P[:, :B] = z                               # p = q: the residual has no mass
    y.fill_(7)
    y[0, 0] = -1
    y[1, 2] = V
    acc, tok, n_new = _run(gpu_lib, y, z, P, 1.0, seed=2, step=0)
    r, t, _, _ = OS.verify(P.cpu().numpy(), z.cpu().numpy(), y.cpu().numpy(), 1.0, 2, 0)
    assert r.tolist() == [0, 2, B] and acc.tolist() == [0, 2, B]
    assert np.array_equal(tok, t)              # the fallback draw is the bonus rule
    assert np.array_equal(n_new, acc + 1)


@pytest.mark.parametrize("batch,B,V,k", [(4, 6, 1003, 5), (3, 16, 151936, 50), (2, 3, 300, 299)])
def test_top_k_verify_matches_oracle(gpu_lib, batch, B, V, k):
    """A top-k proposal: q = 0 outside each draft row's support, candidates
    outside it rejected, the residual equal to p there."""
    y, z, P = synth.verify_round(batch, B, V, seed=k + V, device="cuda")
    for step in range(2):
        lse = gpu_lib.sample(z.reshape(-1, V), 1.0, k, seed=9, step=step)
        y = lse[0].reshape(batch, B).to(torch.int32)          # drafted from the support
        if step == 1:
            y[0, 0] = int(z[0, 0].argmin())                   # outside the support: rejected
        acc, tok, n_new = _run(gpu_lib, y, z, P, 1.0, seed=8, step=step, top_k=k)
        r, _, _ = _compare(acc, tok, n_new, y, z, P, 1.0, 8, step, top_k=k)
        if step == 1:
            assert r[0] == 0 and acc[0] == 0


def test_verify_rejects_bad_arguments(gpu_lib):
    y, z, P = synth.verify_round(2, 3, 100, device="cuda")
    lse = torch.zeros(2, 3, device="cuda")
    with pytest.raises(RuntimeError):
        gpu_lib.verify(P, None, lse, y, 1.0, 0, 0)        # T > 0 needs the draft logits
    with pytest.raises(RuntimeError):
        gpu_lib.verify(P, z, lse, y, -1.0, 0, 0)
    ws = torch.empty(16, dtype=torch.uint8, device="cuda")
    with pytest.raises(RuntimeError):
        gpu_lib.verify(P, z, lse, y, 1.0, 0, 0, workspace=ws)
