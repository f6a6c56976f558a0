"""GPU parity of the mean-pooled summary (the views as the configurations word
them: the last W rows plus strided chunk means): the pooled banks' slot means
against the oracle's running means, the window and boundary bit-exact, and the
drafter's logits over [block; window; pooled slots] against the oracle
forward, for arrivals that cross chunk boundaries and wrap both rings."""
import numpy as np
import pytest
import torch

import synth
from gpu_common import Pair, check_logits, check_views
from oracle import draft as OD

pytestmark = pytest.mark.gpu

MINI_BF16_POOLED = synth.QWEN3_8B.replace(name="mini-bf16-pooled", hidden=512, n_q_heads=8,
                                          n_kv_heads=2, mlp=1024, vocab=5003, n_layers=2,
                                          n_feat_layers=3, window=64, pool_strides=(4, 16),
                                          pool_slots=32)


def run(gpu_lib, s, batch, prefix, chunk, decode=3, ragged=3):
    p = Pair(gpu_lib, s, batch, None)
    if prefix:
        p.prefill(prefix, chunk, ragged=ragged)
    if decode:
        p.decode(decode, s.block + 1, np.random.default_rng(11))
    check_views(p)
    w = synth.make_weights(s, gain_std=0.1, device="cuda")
    dw = gpu_lib.DraftWeights(w)
    anchor = synth.make_anchors(s, batch, device="cuda")
    z = gpu_lib.draft_step(p.views, dw, anchor)
    torch.cuda.synchronize()
    Wt = synth.weights_f64(w)
    a = anchor.cpu().numpy()
    zc = z.cpu().numpy()
    for b in p.seqs:
        check_logits(zc[b], OD.forward(s, Wt, p.ost[b], None, int(a[b])), s)
    assert p.views.status() == 0
    return p


@pytest.mark.parametrize("prefix,chunk", [(0, 1), (3, 3), (70, 33), (300, 128), (2500, 1000)])
def test_pooled_tiny_fp32(gpu_lib, prefix, chunk):
    """Strides 4 and 64, 32 slots each: bank 0 wraps after 128 rows, bank 1
    after 2048."""
    run(gpu_lib, synth.TINY_POOLED, 2, prefix, chunk)


@pytest.mark.parametrize("prefix,chunk", [(5, 5), (150, 64), (700, 300)])
def test_pooled_bf16_mfma(gpu_lib, prefix, chunk):
    """bf16 GQA shape on the matrix-core attention (64 window rows + 2 x 32
    slots = 128 region rows)."""
    run(gpu_lib, MINI_BF16_POOLED, 3, prefix, chunk)


def test_pooled_without_the_window(gpu_lib):
    run(gpu_lib, MINI_BF16_POOLED.replace(drop_views=1), 2, 200, 90)


def test_pooled_slots_track_single_row_updates(gpu_lib):
    """One row per update: every slot passes through every open-chunk state."""
    s = synth.TINY_POOLED.replace(pool_strides=(3, 5))
    p = Pair(gpu_lib, s, 2, None)
    rng = np.random.default_rng(2)
    for step in range(40):
        K, V, h = synth.decode_rows(s, 2, 1, 100 + step, device="cuda")
        p.ingest([int(x) for x in rng.integers(0, 2, 2)], K, V, h)
    check_views(p)


@pytest.mark.slow
def test_pooled_full_size_qwen3_8b(gpu_lib):
    """Qwen3-8B shape with the mean-pooled summary (W 256 + 2 x 256 slots), batch
    16, 8192-row prefix plus a decode update: views of two sequences and their
    logits on a 2048-token vocabulary sample against the oracle."""
    from gpu_common import lazy_weights_f64, row_errors
    s = synth.QWEN3_8B_POOLED
    p = Pair(gpu_lib, s, 16, None, oracle_seqs=[0, 9])
    p.prefill(8192, 4096)
    K, V, h = synth.decode_rows(s, 16, 17, 0, device="cuda")
    p.ingest([17] * 16, K, V, h)
    check_views(p)
    w = synth.make_weights(s, device="cuda")
    dw = gpu_lib.DraftWeights(w, tiled_head=True)
    anchor = synth.make_anchors(s, 16, device="cuda")
    z = gpu_lib.draft_step(p.views, dw, anchor)
    torch.cuda.synchronize()
    idx = np.sort(np.random.default_rng(4).choice(s.vocab, 2048, replace=False))
    Wt = lazy_weights_f64(w)
    a = anchor.cpu().numpy()
    zc = z[:, :, torch.from_numpy(idx).cuda()].cpu().numpy()
    for b in p.seqs:
        ref = OD.forward(s, Wt, p.ost[b], None, int(a[b]), vocab_idx=idx)
        err, cos = row_errors(zc[b], ref)
        assert err.max() <= 2e-2, err.max()
        assert cos.min() >= 0.999, cos.min()
