"""GPU parity of the views update (Sec. 2.2; App. A.2, Eq. 10-11): window
ring, bookkeeping and boundary states bit-exact, summary (eta, m) against the
oracle's incremental fp64 merge."""
import numpy as np
import pytest
import torch

import synth
from gpu_common import Pair, check_views

pytestmark = pytest.mark.gpu

# bf16 with grouped query heads (4 q heads per kv head), two layers
MINI_BF16 = synth.QWEN3_8B.replace(name="mini-bf16", hidden=512, n_q_heads=8, n_kv_heads=2,
                                   mlp=1024, vocab=5003, n_layers=2, n_feat_layers=3,
                                   window=64)


@pytest.mark.parametrize("shape,gscale", [(synth.TINY, 1.0), (synth.TINY, 8.0),
                                          (MINI_BF16, 1.0), (MINI_BF16, 8.0)])
def test_prefill_then_decode(gpu_lib, shape, gscale):
    G = synth.make_G(shape, scale=gscale, device="cuda")
    p = Pair(gpu_lib, shape, 3, G)
    p.prefill(700, 256, ragged=5)          # ragged last chunk, n > W in one update
    check_views(p)
    p.decode(40, shape.block + 1, np.random.default_rng(0))   # includes n = 0 updates
    check_views(p)


def test_short_prefix_partial_window(gpu_lib):
    s = synth.TINY
    p = Pair(gpu_lib, s, 2, synth.make_G(s, device="cuda"))
    p.prefill(9, 9)
    check_views(p)
    p.decode(3, 2, np.random.default_rng(1))
    check_views(p)


def test_empty_update_is_bit_identical(gpu_lib):
    s = MINI_BF16
    p = Pair(gpu_lib, s, 2, synth.make_G(s, device="cuda"))
    p.prefill(100, 100)
    torch.cuda.synchronize()
    before = p.views.arena.clone()
    pos = p.views.pos.clone()
    K, V, h = synth.decode_rows(s, 2, s.block + 1, 0, device="cuda")
    p.views.update(torch.zeros(2, dtype=torch.int32, device="cuda"), K, V, h)
    torch.cuda.synchronize()
    assert torch.equal(before, p.views.arena)
    assert torch.equal(pos, p.views.pos)


def test_out_of_range_count_sets_sticky_flag(gpu_lib):
    s = synth.TINY
    p = Pair(gpu_lib, s, 3, synth.make_G(s, device="cuda"))
    p.prefill(50, 50)
    torch.cuda.synchronize()
    before = p.views.arena.view(3, -1).clone()
    K, V, h = synth.decode_rows(s, 3, 4, 0, device="cuda")
    n = torch.tensor([2, 5, -1], dtype=torch.int32, device="cuda")   # 5 > max_new = 4; -1 < 0
    p.views.update(n, K, V, h)
    assert p.views.status() == gpu_lib.LDR_ERANGE
    after = p.views.arena.view(3, -1)
    assert torch.equal(before[1], after[1]) and torch.equal(before[2], after[2])
    assert not torch.equal(before[0], after[0])
    assert p.views.pos.cpu().tolist() == [52, 50, 50]
    assert p.views.status(clear=True) == gpu_lib.LDR_ERANGE
    assert p.views.status() == gpu_lib.LDR_OK


@pytest.mark.slow
def test_full_size_qwen3_8b_prefill_sampled(gpu_lib):
    """Qwen3-8B shape, batch 16, prefix 32768 ingested in 4096-row chunks, then
    64 decode updates of 17 rows: bookkeeping for all sequences, window and
    summary of two sampled sequences against the oracle."""
    s = synth.QWEN3_8B
    G = synth.make_G(s, device="cuda")
    p = Pair(gpu_lib, s, 16, G, oracle_seqs=[0, 13])
    p.prefill(32768, 4096)
    rng = np.random.default_rng(2)
    for st in range(64):
        K, V, h = synth.decode_rows(s, 16, 17, st, device="cuda")
        p.ingest([17] * 16, K, V, h)
    del rng
    assert p.views.pos.cpu().tolist() == [32768 + 64 * 17] * 16
    check_views(p)
