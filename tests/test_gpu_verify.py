"""GPU parity of speculative verification (Eq. 1-2) against the oracle, fed
the same seeded fp32 logits and candidates.

The acceptance test and the residual draw are decisions taken from fp32
values on the GPU and float64 values in the oracle, so the counts and tokens
must agree exactly wherever the decision has a margin above the fp32 error
(the ratio within 1e-4 relative of u, or a residual key within 1e-3 of the
best, is a near tie); n_new is always r + 1, and bonus tokens (keys that both
sides compute as the same fp32 operations) agree exactly."""
import numpy as np
import pytest
import torch

import synth
from oracle import sample as OS

pytestmark = pytest.mark.gpu

RATIO_TOL = 1e-4
KEY_TOL = 1e-3


def _run(ldr, y, z, P, T, seed, step):
    batch, B, V = z.shape
    lse = None
    if T > 0:
        lse = ldr.sample(z.reshape(-1, V), T, 0, seed=seed + 1, step=step)[1].reshape(batch, B)
    acc, tok, n_new = ldr.verify(P, z if T > 0 else None, lse, y, T, seed, step)
    torch.cuda.synchronize()
    return acc.cpu().numpy(), tok.cpu().numpy(), n_new.cpu().numpy()


def _compare(acc, tok, n_new, y, z, P, T, seed, step, max_ties=1):
    """Counts and tokens against the oracle; returns (oracle r, oracle token,
    indices of the sequences decided without a near tie)."""
    r, t, ratio, u, keys = OS.verify(P.cpu().numpy(), z.cpu().numpy(), y.cpu().numpy(), T,
                                     seed, step, keys=True)
    B = z.shape[1]
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
        k = keys[b]
        if T == 0 or r[b] == B:                 # argmax / bonus keys: the same fp32 values
            assert tok[b] == t[b], (b, tok[b], t[b])
            clean.append(b)
            continue
        gap = k[t[b]] - np.max(np.delete(k, t[b])) if len(k) > 1 else np.inf
        if gap > KEY_TOL:
            assert tok[b] == t[b], (b, tok[b], t[b], gap)
            clean.append(b)
        else:
            ties += 1
            assert k[tok[b]] >= k[t[b]] - KEY_TOL
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
    batch, B, V = 3, 4, 1000
    y, z, P = synth.verify_round(batch, B, V, seed=4, device="cuda")
    P[:, :B] = z                               # p = q: the residual has no mass
    y[0, 0] = -1
    y[1, 2] = V
    acc, tok, n_new = _run(gpu_lib, y, z, P, 1.0, seed=2, step=0)
    r, t, clean = _compare(acc, tok, n_new, y, z, P, 1.0, 2, 0, max_ties=0)
    assert r.tolist() == [0, 2, B] and acc.tolist() == [0, 2, B]
    assert np.array_equal(tok, t)              # the fallback draw is the bonus rule


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
