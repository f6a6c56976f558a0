"""GPU parity of the draft step (Eq. 4, Eq. 6; Sec. 2.3; App. A.1): base
logits of the HIP path against the fp64 oracle forward over the oracle's own
views of the same inputs, plus the structural properties (depends only on
the views, deterministic, t = 0 and partial windows)."""
import numpy as np
import pytest
import torch

import synth
from gpu_common import Pair, check_logits, check_views, lazy_weights_f64, row_errors
from oracle import draft as OD

pytestmark = pytest.mark.gpu

MINI_BF16 = synth.QWEN3_8B.replace(name="mini-bf16", hidden=512, n_q_heads=8, n_kv_heads=2,
                                   mlp=1024, vocab=5003, n_layers=2, n_feat_layers=3,
                                   window=64)


def setup(gpu_lib, shape, batch, prefix, gain_std=0.1, decode=3, tiled_head=False):
    G = synth.make_G(shape, device="cuda")
    p = Pair(gpu_lib, shape, batch, G)
    if prefix:
        p.prefill(prefix, max(prefix // 2, 1), ragged=3)
    if decode:
        p.decode(decode, shape.block + 1, np.random.default_rng(7))
    w = synth.make_weights(shape, gain_std=gain_std, device="cuda")
    dw = gpu_lib.DraftWeights(w, tiled_head=tiled_head)
    anchor = synth.make_anchors(shape, batch, device="cuda")
    return p, w, dw, anchor


def oracle_logits(p, w, anchor, seqs=None, vocab_idx=None, lazy=False):
    Wt = lazy_weights_f64(w) if lazy else synth.weights_f64(w)
    a = anchor.cpu().numpy()
    seqs = p.seqs if seqs is None else seqs
    return {b: OD.forward(p.s, Wt, p.ost[b], p.G64, int(a[b]), vocab_idx=vocab_idx) for b in seqs}


# the Qwen3-32B MLP width: 51200 SwiGLU columns take 128-wide tiles (two rounds
# over the CUs instead of three of 96)
MINI_BF16_MLP32B = MINI_BF16.replace(name="mini-bf16-mlp25600", mlp=25600)


@pytest.mark.parametrize("shape,batch,prefix", [
    (synth.TINY, 1, 2048),     # the fp32 parity configuration
    (synth.TINY, 3, 40),       # partial window (t < W)
    (MINI_BF16, 1, 300),       # bf16, 16 rows: the 16-row GEMM tiles (128 and 96 columns)
    (MINI_BF16, 3, 300),       # bf16, GQA, ragged vocab, 48 rows
    (MINI_BF16, 17, 150),      # bf16, 272 rows: two M tiles, the last ragged
    (MINI_BF16_MLP32B, 16, 100),
])
def test_logits_match_oracle(gpu_lib, shape, batch, prefix):
    p, w, dw, anchor = setup(gpu_lib, shape, batch, prefix)
    z = gpu_lib.draft_step(p.views, dw, anchor)
    torch.cuda.synchronize()
    ref = oracle_logits(p, w, anchor)
    zc = z.cpu().numpy()
    for b in p.seqs:
        check_logits(zc[b], ref[b], shape)


# 90000 tokens: 297 column tiles of 304, more than one round over the 256 CUs,
# the last tile 16 columns wide, its staged weight rows past the padded matrix
MINI_BF16_WIDE_V = MINI_BF16.replace(name="mini-bf16-v90000", vocab=90000)


@pytest.mark.parametrize("shape,batch,prefix", [(MINI_BF16, 5, 300), (MINI_BF16, 17, 150),
                                                (MINI_BF16_WIDE_V, 5, 200)])
def test_tiled_head_matches_oracle_and_row_major(gpu_lib, shape, batch, prefix):
    """The vocabulary head on the tiled copy of lm_head (ldr_tile_matrix),
    used above 64 rows: logits against the oracle, and against the row-major
    head, from which they differ only in the fp32 summation order of the same
    bf16 products. 5 sequences: 80 rows in one ragged M tile; 17 sequences:
    272 rows, two M tiles, the last ragged; V = 5003: a ragged N tile;
    V = 90000: 297 tiles, more workgroups than CUs, a last tile of 16
    columns."""
    s = shape
    p, w, dw, anchor = setup(gpu_lib, s, batch, prefix, tiled_head=True)
    z = gpu_lib.draft_step(p.views, dw, anchor)
    z_rm = gpu_lib.draft_step(p.views, gpu_lib.DraftWeights(w), anchor)
    torch.cuda.synchronize()
    ref = oracle_logits(p, w, anchor)
    zc = z.cpu().numpy()
    for b in p.seqs:
        check_logits(zc[b], ref[b], s)
    scale = z_rm.abs().amax(dim=-1, keepdim=True)
    assert ((z - z_rm).abs() / scale).max().item() <= 1e-4


def test_small_steps_keep_the_row_major_head(gpu_lib):
    """At 64 rows or fewer the head reads lm_head even when a tiled copy is
    given: the logits are bit-identical to the row-major head's."""
    p, w, dw, anchor = setup(gpu_lib, MINI_BF16, 3, 120, tiled_head=True)
    z = gpu_lib.draft_step(p.views, dw, anchor)
    z_rm = gpu_lib.draft_step(p.views, gpu_lib.DraftWeights(w), anchor)
    torch.cuda.synchronize()
    assert torch.equal(z, z_rm)


def test_tile_matrix_layout(gpu_lib):
    """ldr_tile_matrix: column block c / 32 holds all R = 512 (padded) rows of
    its 32 elements one after another, padding rows zero; bit-exact (a pure
    copy)."""
    rows, cols, ld = 300, 96, 104
    g = torch.Generator(device="cuda").manual_seed(5)
    base = torch.randn(rows, ld, device="cuda", generator=g).to(torch.bfloat16)
    m = base[:, :cols]
    t = gpu_lib.tile_matrix(m)
    assert t.numel() * 2 == gpu_lib.tiled_bytes(rows, cols) == 512 * cols * 2
    pad = torch.zeros(512, cols, dtype=torch.bfloat16, device="cuda")
    pad[:rows] = m
    ref = pad.view(512, cols // 32, 32).permute(1, 0, 2).reshape(-1)
    torch.cuda.synchronize()
    assert torch.equal(t.view(torch.int16), ref.view(torch.int16))


def test_tiled_head_rejected_where_unsupported(gpu_lib):
    # fp32 configurations have no tiled head
    p, w, dw, anchor = setup(gpu_lib, synth.TINY, 1, 40, decode=0)
    fake = torch.zeros(gpu_lib.tiled_bytes(synth.TINY.vocab, synth.TINY.hidden) // 2,
                       dtype=torch.bfloat16, device="cuda")
    dw.c.lm_head_tiled = fake.data_ptr()
    with pytest.raises(gpu_lib.LdrError) as e:
        gpu_lib.draft_step(p.views, dw, anchor)
    assert e.value.code == gpu_lib.LDR_EINVAL


@pytest.mark.parametrize("shape", [synth.TINY, MINI_BF16])
def test_empty_views(gpu_lib, shape):
    # t = 0: no window rows, no summary; only the block attends to itself
    p, w, dw, anchor = setup(gpu_lib, shape, 2, 0, decode=0)
    z = gpu_lib.draft_step(p.views, dw, anchor)
    torch.cuda.synchronize()
    ref = oracle_logits(p, w, anchor)
    for b in p.seqs:
        check_logits(z.cpu().numpy()[b], ref[b], shape)


def test_deterministic_and_depends_only_on_views(gpu_lib):
    s = MINI_BF16
    p, w, dw, anchor = setup(gpu_lib, s, 4, 200)
    z1 = gpu_lib.draft_step(p.views, dw, anchor).clone()
    z2 = gpu_lib.draft_step(p.views, dw, anchor).clone()
    torch.cuda.synchronize()
    assert torch.equal(z1, z2)
    # snapshot the arena and positions, move the views on, restore: identical logits
    snap, pos = p.views.arena.clone(), p.views.pos.clone()
    K, V, h = synth.decode_rows(s, 4, s.block + 1, 99, device="cuda")
    p.views.update(torch.full((4,), s.block + 1, dtype=torch.int32, device="cuda"), K, V, h)
    z3 = gpu_lib.draft_step(p.views, dw, anchor).clone()
    torch.cuda.synchronize()
    assert not torch.equal(z1, z3)
    # poison the rows that were just ingested: the draft reads only the views
    K.fill_(float("nan")); V.fill_(float("nan")); h.fill_(float("nan"))
    p.views.arena.copy_(snap)
    p.views.pos.copy_(pos)
    z4 = gpu_lib.draft_step(p.views, dw, anchor)
    torch.cuda.synchronize()
    assert torch.equal(z1, z4)


@pytest.mark.slow
@pytest.mark.parametrize("tiled_head", [True, False])
def test_full_size_qwen3_8b_sampled(gpu_lib, tiled_head):
    """Qwen3-8B shape, batch 16, prefix 32768: the configuration the benchmark
    times (tiled head). Oracle on two sequences, all 16 slots, a 2048-token
    vocabulary sample."""
    s = synth.QWEN3_8B
    G = synth.make_G(s, device="cuda")
    p = Pair(gpu_lib, s, 16, G, oracle_seqs=[0, 11])
    p.prefill(32768, 4096)
    K, V, h = synth.decode_rows(s, 16, 17, 0, device="cuda")
    p.ingest([17] * 16, K, V, h)
    w = synth.make_weights(s, device="cuda")
    dw = gpu_lib.DraftWeights(w, tiled_head=tiled_head)
    anchor = synth.make_anchors(s, 16, device="cuda")
    z = gpu_lib.draft_step(p.views, dw, anchor)
    torch.cuda.synchronize()
    idx = np.sort(np.random.default_rng(3).choice(s.vocab, 2048, replace=False))
    idx = np.concatenate([[0], idx, [s.vocab - 1]])
    ref = oracle_logits(p, w, anchor, vocab_idx=idx, lazy=True)
    zc = z[:, :, torch.from_numpy(idx).cuda()].cpu().numpy()
    for b in p.seqs:
        err, cos = row_errors(zc[b], ref[b])
        assert err.max() <= 2e-2, err.max()
        assert cos.min() >= 0.999, cos.min()


def _sampled_parity(gpu_lib, s, batch, prefix, seqs, tiled_head=True, chunk=4096):
    """Views of `seqs` against the oracle's, then their logits on a 2048-token
    vocabulary sample (plus the first and last token), all B slots."""
    G = synth.make_G(s, device="cuda")
    p = Pair(gpu_lib, s, batch, G, oracle_seqs=seqs)
    p.prefill(prefix, chunk)
    K, V, h = synth.decode_rows(s, batch, s.block + 1, 0, device="cuda")
    p.ingest([s.block + 1] * batch, K, V, h)
    check_views(p)
    w = synth.make_weights(s, device="cuda")
    dw = gpu_lib.DraftWeights(w, tiled_head=tiled_head)
    anchor = synth.make_anchors(s, batch, device="cuda")
    z = gpu_lib.draft_step(p.views, dw, anchor)
    torch.cuda.synchronize()
    assert p.views.status() == 0
    idx = np.sort(np.random.default_rng(5).choice(s.vocab, 2048, replace=False))
    idx = np.concatenate([[0], idx, [s.vocab - 1]])
    ref = oracle_logits(p, w, anchor, vocab_idx=idx, lazy=True)
    zc = z[:, :, torch.from_numpy(idx).cuda()].cpu().numpy()
    for b in p.seqs:
        err, cos = row_errors(zc[b], ref[b])
        assert err.max() <= 2e-2, (b, err.max())
        assert cos.min() >= 0.999, (b, cos.min())


@pytest.mark.slow
def test_full_size_qwen3_32b_sampled(gpu_lib):
    """Qwen3-32B shape (hidden 5120, 64 query heads over 8 kv heads, MLP
    25600), batch 16, prefix 65536: the 32B configuration. Oracle on two
    sequences."""
    _sampled_parity(gpu_lib, synth.QWEN3_32B, 16, 65536, [0, 13])


@pytest.mark.slow
def test_qwen3_8b_batch_64_sampled(gpu_lib):
    """Qwen3-8B shape at 64 sequences, the sweep's largest batch: 1024 rows,
    four row tiles in every GEMM and in the tiled head. Oracle on the first
    and the last sequence."""
    _sampled_parity(gpu_lib, synth.QWEN3_8B, 64, 1000, [0, 63], chunk=500)
