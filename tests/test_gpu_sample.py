"""GPU parity of per-position sampling (Eq. 8): the Gumbel noise of both
levels bit for bit; tokens equal to the oracle's two-level draw from the same
fp32 logits buffer, except where two chunk keys tie within the fp32 error of
the kernel's chunk log-masses (then the GPU's chunk must be such a near tie
and its token that chunk's exact draw; at most one such row per call); lse
and log q within fp32 tolerance."""
import numpy as np
import pytest
import torch

from gpu_common import draw_near_tie
from oracle import sample as OS

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("rows,vocab,stream", [(3, 151936, 0), (37, 1001, 0), (5, 7, 0),
                                               (16, 9496, 3), (3, 257, 3), (2, 100, 1)])
def test_gumbel_noise_is_bit_exact(gpu_lib, rows, vocab, stream):
    g = gpu_lib.gumbel_fill(1234, 9, rows, vocab, noise_stream=stream).cpu().numpy()
    ref = OS.gumbel(1234, 9, np.arange(rows)[:, None], np.arange(vocab)[None, :], stream)
    assert g.dtype == np.float32
    assert np.array_equal(g.view(np.uint32), ref.view(np.uint32))


def _tokens_match(tok, y, z, T, k, seed, step, rows=None):
    """The GPU tokens against the oracle's draw from the same logits: equal, or
    (at most one row) a near tie of the chunk keys within fp32 error."""
    tok = np.asarray(tok).astype(np.int64)
    rows = np.arange(len(y)) if rows is None else rows
    ties = sum(draw_near_tie(z[i], int(y[i]), int(tok[i]), int(rows[i]), T, seed, step, 0.0, k)
               for i in range(len(y)) if tok[i] != y[i])
    assert ties <= 1, ties


def _logits(rows, vocab, seed, scale=1.3):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    return torch.randn(rows, vocab, generator=g, device="cuda") * scale


@pytest.mark.parametrize("rows,vocab,T", [(32, 151936, 1.0), (16, 151936, 0.7),
                                          (300, 5003, 1.0), (9, 2049, 1.7), (4, 3, 1.0)])
def test_tokens_exact_given_the_same_logits(gpu_lib, rows, vocab, T):
    z = _logits(rows, vocab, rows * 7 + vocab)
    tok, lse, logq = gpu_lib.sample(z, T, 0, seed=77, step=5)
    torch.cuda.synchronize()
    zc = z.cpu().numpy()
    y, l, lq = OS.sample(zc, T, 0, 77, 5)
    _tokens_match(tok.cpu().numpy(), y, zc, T, 0, 77, 5)
    np.testing.assert_allclose(lse.cpu().numpy(), l, rtol=2e-6, atol=2e-5)
    np.testing.assert_allclose(logq.cpu().numpy(), lq, rtol=1e-5, atol=2e-4)


def test_greedy_and_ties(gpu_lib):
    z = _logits(50, 151936, 3)
    z[4, 1000] = 50.0
    z[4, 70000] = 50.0          # tie: the lower index wins
    z[7, :] = 0.0               # all equal: token 0
    tok, lse, logq = gpu_lib.sample(z, 0.0, 0, seed=0, step=0)
    torch.cuda.synchronize()
    y, l, lq = OS.sample(z.cpu().numpy(), 0.0, 0, 0, 0)
    assert np.array_equal(tok.cpu().numpy().astype(np.int64), y)
    assert tok[4].item() == 1000 and tok[7].item() == 0
    assert np.array_equal(lse.cpu().numpy(), l.astype(np.float32))
    assert np.all(logq.cpu().numpy() == 0)


def test_steps_and_seeds_change_the_draw(gpu_lib):
    z = torch.zeros(256, 4096, device="cuda")
    a = gpu_lib.sample(z, 1.0, 0, seed=1, step=0)[0].cpu()
    b = gpu_lib.sample(z, 1.0, 0, seed=1, step=1)[0].cpu()
    c = gpu_lib.sample(z, 1.0, 0, seed=2, step=0)[0].cpu()
    assert (a != b).float().mean() > 0.9 and (a != c).float().mean() > 0.9
    # uniform logits: every token is equally likely, lse = log V exactly in exact arithmetic
    lse = gpu_lib.sample(z, 1.0, 0, seed=1, step=0)[1].cpu().numpy()
    np.testing.assert_allclose(lse, np.log(4096.0), rtol=1e-6)


def _check_sample(gpu_lib, z, T, k, seed, step):
    tok, lse, logq = gpu_lib.sample(z, T, k, seed=seed, step=step)
    torch.cuda.synchronize()
    zc = z.cpu().numpy()
    y, l, lq = OS.sample(zc, T, k, seed, step)
    _tokens_match(tok.cpu().numpy(), y, zc, T, k, seed, step)
    np.testing.assert_allclose(lse.cpu().numpy(), l, rtol=2e-6, atol=2e-5)
    np.testing.assert_allclose(logq.cpu().numpy(), lq, rtol=1e-5, atol=2e-4)
    return tok.cpu().numpy()


@pytest.mark.parametrize("rows,vocab,T,k", [(16, 151936, 1.0, 50), (9, 2049, 0.7, 1),
                                            (33, 5003, 1.0, 5002), (8, 1001, 1.3, 1000),
                                            (4, 3, 1.0, 2), (64, 4096, 1.0, 7)])
def test_top_k_tokens_exact(gpu_lib, rows, vocab, T, k):
    z = _logits(rows, vocab, rows * 11 + vocab + k)
    tok = _check_sample(gpu_lib, z, T, k, seed=91, step=3)
    for r in range(rows):  # every token is inside the row's top-k support
        assert tok[r] in set(OS.support(z[r].cpu().numpy(), k).tolist())


def test_top_k_ties_at_the_boundary(gpu_lib):
    # few distinct values: the k-th value is shared by many tokens, and the
    # lowest indices among them are inside
    z = torch.round(_logits(12, 20011, 5) * 2.0) / 2.0
    z[3, :] = 0.25                                  # all equal: the first k tokens
    z[5, ::2] = -0.0                                # -0 and +0 compare equal
    z[5, 1::2] = 0.0
    z[5, 17] = 1.0
    for k in (1, 40, 333, 20010):
        _check_sample(gpu_lib, z, 1.0, k, seed=k, step=1)


def test_top_k_at_least_vocab_is_the_full_support(gpu_lib):
    z = _logits(20, 3001, 8)
    a = gpu_lib.sample(z, 1.0, 0, seed=4, step=2)
    b = gpu_lib.sample(z, 1.0, 3001, seed=4, step=2)
    c = gpu_lib.sample(z, 1.0, 10**6, seed=4, step=2)
    for x, y in ((a, b), (a, c)):
        assert torch.equal(x[0], y[0]) and torch.equal(x[1], y[1])


@pytest.mark.parametrize("T", [1.0, 0.6])
def test_nan_logit_leaves_its_chunk_out(gpu_lib, T):
    """A NaN logit makes its 16-token chunk's log-mass NaN, which the chunk
    draw leaves out as it does a chunk of -inf logits: tokens, lse and log q
    equal those of the same rows with that chunk at -inf, bit for bit, and no
    token comes from it (NaN logits are outside the sampler's contract; this
    pins what the kernels do with them)."""
    rows, V, c = 12, 5003, 7
    g = torch.Generator(device="cuda").manual_seed(3)
    z = torch.randn(rows, V, device="cuda", generator=g) * 3
    z[:, c * 16:(c + 1) * 16] += 6.0          # a chunk that would often win
    zn = z.clone()
    zn[:, c * 16 + 5] = float("nan")
    zi = z.clone()
    zi[:, c * 16:(c + 1) * 16] = float("-inf")
    a = gpu_lib.sample(zn, T, 0, 11, 2)
    b = gpu_lib.sample(zi, T, 0, 11, 2)
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x, y)
    tok = a[0]
    assert not torch.any((tok >= c * 16) & (tok < (c + 1) * 16))
    ref = gpu_lib.sample(z, T, 0, 11, 2)[0]    # without the NaN the chunk is drawn
    assert torch.any((ref >= c * 16) & (ref < (c + 1) * 16))


def test_negative_top_k_is_rejected(gpu_lib):
    z = _logits(2, 100, 1)
    with pytest.raises(gpu_lib.LdrError):
        gpu_lib.sample(z, 1.0, -1, seed=0, step=0)


# ---- Markov-corrected sampling (Eq. 7-8) ----------------------------------------------------

def _markov_case(batch, B, vocab, rank, dtype, seed, scale=0.4):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    z0 = torch.randn(batch, B, vocab, generator=g, device="cuda") * 1.3
    E = (torch.randn(vocab, rank, generator=g, device="cuda") * scale).to(dtype)
    W = (torch.randn(vocab, rank, generator=g, device="cuda") * scale).to(dtype)
    a = torch.randint(0, vocab, (batch,), generator=g, device="cuda", dtype=torch.int32)
    return z0, a, E, W


@pytest.mark.parametrize("batch,B,vocab,rank,dtype,T,k", [
    (4, 8, 151936, 64, torch.bfloat16, 1.0, 0),     # the Qwen3 vocabulary
    (3, 5, 1001, 8, torch.float32, 0.7, 0),         # fp32 correction, ragged vocab
    (18, 3, 5003, 16, torch.bfloat16, 1.0, 40),     # more sequences than one LDS batch, top-k
    (2, 6, 4099, 32, torch.bfloat16, 0.0, 0),       # greedy
])
def test_markov_matches_oracle(gpu_lib, batch, B, vocab, rank, dtype, T, k):
    """Corrected logits bit for bit, tokens exactly, lse and log q within fp32
    tolerance, against the oracle's sequential sampling from the same base
    logits, anchors and correction weights (a chunk-key near tie would change
    every later position of its sequence; the chance at these sizes is about
    1e-3 per run)."""
    z0, a, E, W = _markov_case(batch, B, vocab, rank, dtype, batch * 31 + vocab + rank)
    z0_host = z0.cpu().numpy()
    z = z0.clone()
    tok, lse, logq = gpu_lib.sample_markov(z, a, E, W, T, k, seed=13, step=4)
    torch.cuda.synchronize()
    y, l, lq, zc = OS.sample_markov(z0_host, a.cpu().numpy(), E.float().cpu().numpy(),
                                    W.float().cpu().numpy(), T, k, 13, 4)
    assert np.array_equal(z.cpu().numpy().view(np.uint32), zc.view(np.uint32))
    assert np.array_equal(tok.cpu().numpy().astype(np.int64), y)
    np.testing.assert_allclose(lse.cpu().numpy(), l, rtol=2e-6, atol=2e-5)
    np.testing.assert_allclose(logq.cpu().numpy(), lq, rtol=1e-5, atol=2e-4)


def test_markov_without_correction_is_ldr_sample(gpu_lib):
    """W_c = 0 leaves the logits unchanged and draws what ldr_sample draws on
    the [batch * B][V] rows."""
    z0, a, E, W = _markov_case(5, 4, 4096, 8, torch.bfloat16, 3)
    z = z0.clone()
    tok, lse, logq = gpu_lib.sample_markov(z, a, E, torch.zeros_like(W), 1.0, 0, seed=2, step=8)
    tok1, lse1, logq1 = gpu_lib.sample(z0.view(-1, 4096), 1.0, 0, seed=2, step=8)
    torch.cuda.synchronize()
    assert torch.equal(z, z0)
    assert torch.equal(tok.view(-1), tok1) and torch.equal(lse.view(-1), lse1)
    assert torch.equal(logq.view(-1), logq1)


def test_markov_rejects_bad_arguments(gpu_lib):
    z0, a, E, W = _markov_case(2, 2, 512, 8, torch.bfloat16, 1)
    for kw in ({"E": E[:, :6].contiguous(), "W": W[:, :6].contiguous()},   # rank % 8
               {"k": -1}):
        with pytest.raises(gpu_lib.LdrError) as e:
            gpu_lib.sample_markov(z0.clone(), a, kw.get("E", E), kw.get("W", W), 1.0,
                                  kw.get("k", 0), seed=0, step=0)
        assert e.value.code == gpu_lib.LDR_EINVAL
