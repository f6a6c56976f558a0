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
from gpu_common import (Pair, check_logits, check_views, draw_near_tie, residual_decision,
                        row_errors)
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


MINI_BF16 = synth.QWEN3_8B.replace(name="mini-bf16", hidden=512, n_q_heads=8, n_kv_heads=2,
                                   mlp=1024, vocab=5003, n_layers=2, n_feat_layers=3,
                                   window=64)


def test_bf16_rounds_replayed_by_the_oracle(gpu_lib):
    """bf16 closed rounds (hidden 512, 8 query heads over 2 kv heads, vocab
    5003, block 16), 4 sequences, 5 rounds at T = 1: the GPU closes every
    round on the device (draft step -> sampling -> verification -> views
    update by r + 1, the emitted token the next anchor). The oracle replays
    each round from its own views: its logits within the bf16 tolerance of the
    GPU's; every GPU token the oracle's own two-level draw or a near tie of it
    (chunk keys, then token keys, within twice the row's logit error); the GPU's
    acceptance count equal to the oracle's on the GPU's candidates unless the
    deciding ratio is within the logit error of u; the emitted token the
    oracle's unless a near tie of the residual or bonus draw. The oracle's
    views then take the GPU's r + 1 rows and stay equal to the GPU's. The rate
    of GPU tokens that differ from the oracle's own draws is bounded."""
    s, batch, rounds, T = MINI_BF16, 4, 5, 1.0
    B, V = s.block, s.vocab
    G = synth.make_G(s, device="cuda")
    p = Pair(gpu_lib, s, batch, G)
    p.prefill(300, 150, ragged=7)
    w = synth.make_weights(s, gain_std=0.1, device="cuda")
    dw = gpu_lib.DraftWeights(w)
    Wt = synth.weights_f64(w)
    anchor = synth.make_anchors(s, batch, device="cuda")
    mism = ties = 0
    for rnd in range(rounds):
        a = anchor.cpu().numpy().astype(np.int64)
        z = gpu_lib.draft_step(p.views, dw, anchor)
        y, lse, _ = gpu_lib.sample(z.reshape(-1, V), T, 0, seed=21, step=rnd)
        noise = synth.normal((batch, B + 1, V), 1.0, 900 + rnd, device="cuda")
        P = torch.cat([z + 0.3 * noise[:, :B], 2.0 * noise[:, B:]], dim=1).contiguous()
        acc, tok, n_new = gpu_lib.verify(P, z, lse.reshape(batch, B), y.reshape(batch, B), T,
                                         33, rnd)
        K, Vr, h = synth.decode_rows(s, batch, B + 1, rnd, device="cuda")
        p.views.update(n_new, K, Vr, h)
        anchor = tok
        torch.cuda.synchronize()
        zg, yg = z.cpu().numpy(), y.cpu().numpy().reshape(batch, B)
        accg, tokg = acc.cpu().numpy(), tok.cpu().numpy()
        z_o = np.stack([OD.forward(s, Wt, p.ost[b], p.G64, int(a[b]))
                        for b in range(batch)]).astype(np.float32)
        err = np.array([np.abs(zg[b] - z_o[b]).max(axis=-1) for b in range(batch)])   # [b][i]
        for b in range(batch):
            check_logits(zg[b], z_o[b], s)
        # tokens: the oracle's own draw, or a near tie of it
        y_o, _, _ = OS.sample(z_o.reshape(-1, V), T, 0, 21, rnd)
        y_o = y_o.reshape(batch, B)
        for b in range(batch):
            for i in range(B):
                mism += draw_near_tie(z_o[b, i], int(y_o[b, i]), int(yg[b, i]), b * B + i, T,
                                      21, rnd, err[b, i] / T)
        # verification of the GPU's candidates against the oracle's own logits
        nz = noise.cpu().numpy()
        P_o = np.concatenate([z_o + np.float32(0.3) * nz[:, :B], np.float32(2.0) * nz[:, B:]],
                             axis=1)
        r_o, t_o, ratio, u, det = OS.verify(P_o, z_o, yg, T, 33, rnd, detail=True)
        for b in range(batch):
            e = 2 * err[b].max() / T            # log-ratio error bound: both lse and the logit
            n = min(int(max(r_o[b], accg[b])) + 1, B)
            lr = np.log(np.maximum(ratio[b, :n], 1e-300))
            near = np.abs(np.log(u[b, :n]) - lr) <= e + 1e-6
            if accg[b] != r_o[b]:
                first = min(int(accg[b]), int(r_o[b]))
                assert near[first], (rnd, b, accg[b], r_o[b])
                ties += 1
                continue
            if np.any(near):
                ties += 1
                continue
            if r_o[b] == B:                      # bonus row: the same fp32 noise logits
                assert tokg[b] == t_o[b], (rnd, b)
                continue
            g = OS.verify_gumbel(33, rnd, b, np.arange(V))
            bonus_tok = int(np.argmax(P_o[b, r_o[b]] / np.float32(T) + g))
            clean, valid = residual_decision(det[b], bonus_tok, float(np.expm1(2 * e)))
            if clean:
                assert tokg[b] == t_o[b], (rnd, b, tokg[b], t_o[b])
            else:
                ties += 1
                assert int(tokg[b]) in valid, (rnd, b)
        # the oracle's views take the rows the GPU committed
        for b in range(batch):
            nb = int(accg[b]) + 1
            p.ost[b] = OV.update(s, p.ost[b], p.G64, synth.to_f64(K[b, :nb]),
                                 synth.to_f64(Vr[b, :nb]), synth.to_f64(h[b]))
        check_views(p)
    rate = mism / (rounds * batch * B)
    print(f"bf16 rounds: token mismatch rate {rate:.4f}, near-tie verification decisions {ties}")
    assert rate <= 0.1 and ties <= rounds * batch // 2
    assert p.views.status() == 0
