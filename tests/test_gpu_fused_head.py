"""GPU parity of ldr_draft_step_sample: the draft step followed by sampling of
every position. Greedy steps take the first argmax in the vocabulary head's
epilogue: the logits it writes are ldr_draft_step's bit for bit, and its
tokens, lse and log q are the separate sampler's at T = 0 on those logits
(the separate sampler is itself compared with the oracle in
test_gpu_sample.py); without the logits it draws the same tokens. Sampled
steps form the 16-token chunk log-masses in the head's epilogue and then run
the sampler's chunk draw: logits, tokens, lse and log q are the separate
calls' bit for bit (lse sums every chunk's log-mass, so it is equal only if
each of them is)."""
import numpy as np
import pytest
import torch

import synth
from gpu_common import Pair
from oracle import draft as OD
from oracle import sample as OS

pytestmark = pytest.mark.gpu

MINI_BF16 = synth.QWEN3_8B.replace(name="mini-bf16", hidden=512, n_q_heads=8, n_kv_heads=2,
                                   mlp=1024, vocab=5003, n_layers=2, n_feat_layers=3,
                                   window=64)


def setup(gpu_lib, shape, batch, prefix):
    G = synth.make_G(shape, device="cuda")
    p = Pair(gpu_lib, shape, batch, G, oracle_seqs=[])
    p.prefill(prefix, max(prefix // 2, 1), ragged=2)
    w = synth.make_weights(shape, gain_std=0.1, device="cuda")
    return p, gpu_lib.DraftWeights(w, tiled_head=True), synth.make_anchors(shape, batch,
                                                                           device="cuda")


def check(gpu_lib, shape, batch, prefix, T, seed=13, step=4):
    p, dw, anchor = setup(gpu_lib, shape, batch, prefix)
    z_ref = gpu_lib.draft_step(p.views, dw, anchor)
    V = shape.vocab
    tok_ref, lse_ref, logq_ref = gpu_lib.sample(z_ref.view(-1, V), T, 0, seed, step)
    z, tok, lse, logq = gpu_lib.draft_step_sample(p.views, dw, anchor, T, seed, step)
    torch.cuda.synchronize()
    assert torch.equal(z, z_ref)                                # the same head, the same logits
    assert torch.equal(tok.view(-1), tok_ref)                   # the same keys
    np.testing.assert_allclose(lse.view(-1).cpu().numpy(), lse_ref.cpu().numpy(),
                               rtol=2e-6, atol=2e-5)
    np.testing.assert_allclose(logq.view(-1).cpu().numpy(), logq_ref.cpu().numpy(),
                               rtol=1e-5, atol=2e-4)
    if T == 0.0:     # the fused greedy head: bit-exact, and the logits are optional
        assert torch.equal(lse.view(-1), lse_ref) and torch.all(logq == 0)
        _, tok2, lse2, _ = gpu_lib.draft_step_sample(p.views, dw, anchor, T, seed, step,
                                                     logits=None)
        torch.cuda.synchronize()
        assert torch.equal(tok2, tok) and torch.equal(lse2, lse)
    else:            # sampled steps need the logits
        with pytest.raises(RuntimeError):
            gpu_lib.draft_step_sample(p.views, dw, anchor, T, seed, step, logits=None)
    return tok


@pytest.mark.parametrize("batch,T", [(5, 0.0), (17, 0.0), (9, 0.0), (17, 1.0), (5, 0.7)])
def test_draft_step_sample_matches_separate_sampler(gpu_lib, batch, T):
    """5 x 16 = 80 rows (one ragged row tile), 17 x 16 = 272 rows (two, the
    last ragged); vocabulary 5003 (a ragged last column tile)."""
    check(gpu_lib, MINI_BF16, batch, 120, T)


def test_fused_greedy_tokens_against_the_oracle(gpu_lib):
    """The fused greedy head against the oracle's own forward and argmax (the
    oracle never sees a GPU value): the logits agree to 2e-2 of a row's
    largest magnitude, so a GPU token must be the oracle's wherever the
    oracle's two best logits are further apart than twice that, and otherwise
    within it of the oracle's best; lse at T = 0 is the row's largest logit."""
    s, batch = MINI_BF16, 5
    G = synth.make_G(s, device="cuda")
    p = Pair(gpu_lib, s, batch, G)
    p.prefill(120, 60, ragged=2)
    w = synth.make_weights(s, gain_std=0.1, device="cuda")
    dw = gpu_lib.DraftWeights(w, tiled_head=True)
    anchor = synth.make_anchors(s, batch, device="cuda")
    _, tok, lse, logq = gpu_lib.draft_step_sample(p.views, dw, anchor, 0.0, 0, 0, logits=None)
    torch.cuda.synchronize()
    tok, lse = tok.cpu().numpy(), lse.cpu().numpy()
    assert np.all(logq.cpu().numpy() == 0)
    Wt = synth.weights_f64(w)
    a = anchor.cpu().numpy()
    exact = 0
    for b in p.seqs:
        ref = OD.forward(s, Wt, p.ost[b], p.G64, int(a[b]))
        y, top, _ = OS.sample(ref.astype(np.float32), 0.0, 0, 0, 0)
        scale = np.abs(ref).max(axis=1)
        for i in range(s.block):
            tol = 2e-2 * scale[i]
            second = np.max(np.delete(ref[i], y[i]))
            if ref[i, y[i]] - second > 2 * tol:
                assert tok[b, i] == y[i], (b, i, tok[b, i], y[i])
                exact += 1
            else:
                assert ref[i, tok[b, i]] >= ref[i, y[i]] - 2 * tol, (b, i)
            assert abs(lse[b, i] - top[i]) <= tol, (b, i, lse[b, i], top[i])
    assert exact >= 10, exact                   # rows with a clear winner were checked


def test_fused_greedy_head_ties_and_full_size(gpu_lib):
    """Qwen3-8B shape, batch 16: 500 column tiles of the 151936-token head."""
    tok = check(gpu_lib, synth.QWEN3_8B, 16, 300, 0.0)
    assert len(set(tok.view(-1).tolist())) > 1


def test_fused_greedy_head_lowest_index_on_ties(gpu_lib):
    """Two equal largest logits in different column tiles: the lower token,
    as the separate sampler picks it (a zero vocabulary head makes every logit
    of a row equal: token 0)."""
    s = MINI_BF16
    p, dw, anchor = setup(gpu_lib, s, 5, 40)
    w = dict(dw.w)
    w["lm_head"] = torch.zeros_like(w["lm_head"])
    dz = gpu_lib.DraftWeights(w, tiled_head=True)
    _, tok, lse, _ = gpu_lib.draft_step_sample(p.views, dz, anchor, 0.0, 0, 0, logits=None)
    torch.cuda.synchronize()
    assert torch.all(tok == 0) and torch.all(lse == 0)


def test_small_steps_take_the_separate_sampler(gpu_lib):
    """At 64 rows or fewer the head reads the row-major weight: the step then
    runs the separate sampler, which needs the logits."""
    p, dw, anchor = setup(gpu_lib, MINI_BF16, 2, 50)
    z_ref = gpu_lib.draft_step(p.views, dw, anchor)
    tok_ref = gpu_lib.sample(z_ref.view(-1, MINI_BF16.vocab), 1.0, 0, 3, 1)[0]
    z, tok, _, _ = gpu_lib.draft_step_sample(p.views, dw, anchor, 1.0, 3, 1)
    torch.cuda.synchronize()
    assert torch.equal(z, z_ref) and torch.equal(tok.view(-1), tok_ref)
    with pytest.raises(RuntimeError):
        gpu_lib.draft_step_sample(p.views, dw, anchor, 1.0, 3, 1, logits=None)


MINI_WIDE = MINI_BF16.replace(name="mini-bf16-v70000", vocab=70000)
MINI_WIDE_RAGGED = MINI_BF16.replace(name="mini-bf16-v70020", vocab=70020)


@pytest.mark.parametrize("T", [1.0, 0.9, 0.0])
def test_last_tile_ends_inside_a_wave_and_a_chunk(gpu_lib, T):
    """Vocabulary 70020 (a multiple of 4, so the logits rows start on 16
    bytes): the last column tile holds 100 tokens, so its second wave's 80
    columns end inside a 16-token chunk (tokens 96 .. 99 of the tile, the rest
    past the vocabulary), and its last two waves hold no token at all."""
    tok = check(gpu_lib, MINI_WIDE_RAGGED, 9, 120, T)
    assert len(set(tok.view(-1).tolist())) > 1


@pytest.mark.parametrize("batch,T", [(5, 1.0), (16, 0.8)])
def test_sampled_step_matches_the_separate_calls(gpu_lib, batch, T):
    """Vocabulary 70000: 231 column tiles of 304. Logits, tokens, lse and
    log q equal the separate ldr_draft_step + ldr_sample bit for bit, over
    several calls in a row."""
    p, dw, anchor = setup(gpu_lib, MINI_WIDE, batch, 120)
    V = MINI_WIDE.vocab
    for step in range(3):
        z_ref = gpu_lib.draft_step(p.views, dw, anchor)
        tok_ref, lse_ref, logq_ref = gpu_lib.sample(z_ref.view(-1, V), T, 0, 21, step)
        z, tok, lse, logq = gpu_lib.draft_step_sample(p.views, dw, anchor, T, 21, step)
        torch.cuda.synchronize()
        assert torch.equal(z, z_ref)
        assert torch.equal(tok.view(-1), tok_ref)
        assert torch.equal(lse.view(-1), lse_ref) and torch.equal(logq.view(-1), logq_ref)
        assert len(set(tok.view(-1).tolist())) > 1


def test_nan_logit_in_the_fused_head(gpu_lib):
    """A NaN row of the vocabulary head (token 117, chunk 7) gives every row a
    NaN logit: the head's chunk log-mass of that chunk is NaN like the
    log-mass pass's, so the sampled step still equals the separate calls bit
    for bit (logits compared as bits) and never draws from that chunk."""
    p, dw, anchor = setup(gpu_lib, MINI_WIDE, 5, 120)
    w = dict(dw.w)
    head = w["lm_head"].clone()
    head[117] = float("nan")
    w["lm_head"] = head
    dn = gpu_lib.DraftWeights(w, tiled_head=True)
    V = MINI_WIDE.vocab
    z_ref = gpu_lib.draft_step(p.views, dn, anchor)
    ref = gpu_lib.sample(z_ref.view(-1, V), 1.0, 0, 21, 1)
    z, tok, lse, logq = gpu_lib.draft_step_sample(p.views, dn, anchor, 1.0, 21, 1)
    torch.cuda.synchronize()
    assert torch.equal(z.view(torch.int32), z_ref.view(torch.int32))
    assert torch.isnan(z[..., 117]).all()
    for a, b in zip((tok, lse, logq), ref):
        assert torch.equal(a.view(-1), b)
    assert not torch.any((tok >= 112) & (tok < 128))


@pytest.mark.slow
def test_sampled_step_full_size(gpu_lib):
    """Qwen3-8B shape, batch 16, T = 1: the benchmarked call (500 column
    tiles), bit for bit against the separate calls."""
    p, dw, anchor = setup(gpu_lib, synth.QWEN3_8B, 16, 300)
    V = synth.QWEN3_8B.vocab
    z_ref = gpu_lib.draft_step(p.views, dw, anchor)
    ref = gpu_lib.sample(z_ref.view(-1, V), 1.0, 0, 5, 9)
    z, tok, lse, logq = gpu_lib.draft_step_sample(p.views, dw, anchor, 1.0, 5, 9)
    torch.cuda.synchronize()
    assert torch.equal(z, z_ref)
    for a, b in zip((tok, lse, logq), ref):
        assert torch.equal(a.view(-1), b)
