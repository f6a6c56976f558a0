"""GPU parity of the ablation variants (Sec. 3.4, App. D.3): drafters built
without the recent window, the global summary or the boundary state keep
only their other views (bit-exact copies, summary within tolerance) and their
logits follow the oracle's variant forward at the drafting step's tolerance."""
import numpy as np
import pytest
import torch

import synth
from gpu_common import Pair, check_logits, check_views
from oracle import draft as OD

pytestmark = pytest.mark.gpu

MINI_BF16 = synth.QWEN3_8B.replace(name="mini-bf16", hidden=512, n_q_heads=8, n_kv_heads=2,
                                   mlp=1024, vocab=5003, n_layers=2, n_feat_layers=3,
                                   window=64)


@pytest.mark.parametrize("drop", [1, 2, 4, 3])
@pytest.mark.parametrize("shape,batch,prefix", [(synth.TINY, 2, 150), (MINI_BF16, 3, 300)])
def test_variant_matches_oracle(gpu_lib, shape, batch, prefix, drop):
    s = shape.replace(drop_views=drop)
    G = synth.make_G(s, device="cuda")
    p = Pair(gpu_lib, s, batch, G)
    p.prefill(prefix, max(prefix // 2, 1), ragged=3)
    p.decode(2, s.block + 1, np.random.default_rng(5))
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
        ref = OD.forward(s, Wt, p.ost[b], p.G64, int(a[b]))
        check_logits(zc[b], ref, s)
    assert p.views.status() == 0


def test_variants_differ_from_the_full_drafter(gpu_lib):
    """The same inputs through the full drafter and each variant give different
    logits (every view reaches the output)."""
    s0 = MINI_BF16
    out = {}
    for drop in (0, 1, 2, 4):
        s = s0.replace(drop_views=drop)
        G = synth.make_G(s, device="cuda")
        p = Pair(gpu_lib, s, 2, G)
        p.prefill(200, 100)
        dw = gpu_lib.DraftWeights(synth.make_weights(s, gain_std=0.1, device="cuda"))
        out[drop] = gpu_lib.draft_step(p.views, dw, synth.make_anchors(s, 2, device="cuda")).cpu()
    for drop in (1, 2, 4):
        assert (out[drop] - out[0]).abs().max() > 1e-3, drop


def test_summary_queries_optional_only_without_the_summary(gpu_lib):
    s = MINI_BF16.replace(drop_views=2)
    v = gpu_lib.Views(s, 2, None).init()          # no G: accepted
    torch.cuda.synchronize()
    assert v.status() == 0
    with pytest.raises(RuntimeError):
        gpu_lib.Views(MINI_BF16, 2, None).init()  # the full drafter needs G
