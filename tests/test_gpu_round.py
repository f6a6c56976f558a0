"""A closed drafting round on the GPU against the oracle (Eq. 1-2, Eq. 4, Eq. 8;
Sec. 2.3): draft step, sampling, verification against a synthetic target and
the views update by the r + 1 rows the round commits, with the emitted token
as the next anchor. The GPU side keeps every value on the device between the
calls (n_new and the anchor go from ldr_verify straight into the next views
update and draft step); the oracle runs the same loop on its own values. The
target's logits are the round's draft logits plus seeded noise on each side,
with a seeded last row, so that acceptance lengths vary."""
import numpy as np
import pytest
import torch

import synth
from gpu_common import Pair, check_logits, check_views
from oracle import draft as OD
from oracle import sample as OS
from oracle import views as OV

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("T", [1.0, 0.0])
def test_rounds_close_the_loop(gpu_lib, T):
    s, batch, rounds = synth.TINY, 3, 4
    B, V = s.block, s.vocab
    G = synth.make_G(s, device="cuda")
    p = Pair(gpu_lib, s, batch, G)
    p.prefill(150, 64, ragged=5)
    w = synth.make_weights(s, gain_std=0.1, device="cuda")
    dw = gpu_lib.DraftWeights(w)
    Wt = synth.weights_f64(w)
    anchor = synth.make_anchors(s, batch, device="cuda")
    anchor_o = anchor.cpu().numpy().astype(np.int64)
    seen = set()
    for rnd in range(rounds):
        # GPU: every value stays on the device
        z = gpu_lib.draft_step(p.views, dw, anchor)
        y, lse, _ = gpu_lib.sample(z.reshape(-1, V), T, 0, seed=21, step=rnd)
        noise = synth.normal((batch, B + 1, V), 1.0, 700 + rnd, device="cuda")
        P = torch.cat([z + 0.3 * noise[:, :B], 2.0 * noise[:, B:]], dim=1).contiguous()
        acc, tok, n_new = gpu_lib.verify(P, z if T > 0 else None, lse.reshape(batch, B) if T > 0
                                         else None, y.reshape(batch, B), T, 33, rnd)
        K, Vr, h = synth.decode_rows(s, batch, B + 1, rnd, device="cuda")
        p.views.update(n_new, K, Vr, h)
        anchor = tok
        # oracle: its own logits, tokens, verification and views
        z_o = np.stack([OD.forward(s, Wt, p.ost[b], p.G64, int(anchor_o[b]))
                        for b in range(batch)]).astype(np.float32)
        y_o, _, _ = OS.sample(z_o.reshape(-1, V), T, 0, 21, rnd)
        nz = noise.cpu().numpy()
        P_o = np.concatenate([z_o + np.float32(0.3) * nz[:, :B], np.float32(2.0) * nz[:, B:]],
                             axis=1)
        r_o, t_o, _, _ = OS.verify(P_o, z_o, y_o.reshape(batch, B), T, 33, rnd)
        for b in range(batch):
            n = int(r_o[b]) + 1
            p.ost[b] = OV.update(s, p.ost[b], p.G64, synth.to_f64(K[b, :n]),
                                 synth.to_f64(Vr[b, :n]), synth.to_f64(h[b]))
        anchor_o = t_o
        # the two rounds agree
        torch.cuda.synchronize()
        for b in range(batch):
            check_logits(z[b].cpu().numpy(), z_o[b], s)
        assert np.array_equal(y.cpu().numpy().astype(np.int64), y_o)
        assert np.array_equal(acc.cpu().numpy(), r_o), (rnd, acc.cpu().numpy(), r_o)
        assert np.array_equal(n_new.cpu().numpy(), r_o + 1)
        assert np.array_equal(tok.cpu().numpy(), t_o)
        seen.update(r_o.tolist())
        check_views(p)
    assert p.views.status() == 0
    if T > 0:
        assert len(seen) > 2, seen        # the rounds commit different numbers of rows
