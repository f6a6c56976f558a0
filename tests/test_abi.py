"""Host-side checks of libldr.so that need no GPU: every symbol that
include/ldr.h declares is exported, the state-size and layout formulas, the
configuration checks and the synchronous argument validation."""
import ctypes
import os
import re

import pytest

import synth
from oracle import views as oviews

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def L():
    from paper_2609_37029_amd import ldr
    if not os.path.exists(ldr.LIB_PATH):
        pytest.fail("libldr.so is not built (python -m paper_2609_37029_amd.build)")
    return ldr


def declared_functions():
    src = open(os.path.join(ROOT, "include", "ldr.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(ldr_[a-z_]+)\s*\(", src)))


def test_every_declared_symbol_is_exported(L):
    names = declared_functions()
    assert len(names) >= 14
    lib = ctypes.CDLL(L.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n


@pytest.mark.parametrize("shape,expected", [(synth.QWEN3_8B, 6_604_800),
                                            (synth.QWEN3_32B, 7_936_000),
                                            (synth.TINY, 150_784)])
def test_state_bytes(L, shape, expected):
    assert L.state_bytes(shape) == expected == oviews.state_bytes(shape)
    assert L.stride_bytes(shape) % 256 == 0 and L.stride_bytes(shape) >= expected


def test_layout_regions(L):
    s = synth.QWEN3_8B
    off = L.layout(s)
    win = s.n_layers * s.n_kv_heads * s.window * s.head_dim * 2
    assert off["kw"] == 0 and off["vw"] == win and off["m"] == 2 * win
    assert off["eta"] - off["m"] == s.n_layers * s.n_q_heads * s.summary * s.head_dim * 4
    assert off["h"] - off["eta"] == s.n_layers * s.n_q_heads * s.summary * 4
    assert all(v % 256 == 0 for v in off.values())


def test_config_check(L):
    good = L.config(synth.QWEN3_8B)
    assert L.lib().ldr_config_check(ctypes.byref(good)) == L.LDR_OK
    bad = [dict(n_kv_heads=7), dict(head_dim=96), dict(block=17), dict(block=0), dict(dtype=5),
           dict(hidden=4000), dict(window=0), dict(rms_eps=0.0), dict(mlp=100)]
    for kw in bad:
        c = L.config(synth.QWEN3_8B)
        for k, v in kw.items():
            setattr(c, k, v)
        assert L.lib().ldr_config_check(ctypes.byref(c)) == L.LDR_EINVAL, kw
        assert L.lib().ldr_views_state_bytes(ctypes.byref(c)) == 0


def test_workspace_grows_with_batch(L):
    s = synth.QWEN3_8B
    sizes = [L.workspace_bytes(s, b) for b in (1, 16, 64)]
    assert 0 < sizes[0] < sizes[1] < sizes[2]
    assert L.workspace_bytes(s, 0) == 0


def test_host_validation_needs_no_gpu(L):
    lib = L.lib()
    h = ctypes.c_void_p()
    cfg = L.config(synth.TINY)
    # null arena / pos / G: rejected before any device call
    assert lib.ldr_views_init(ctypes.byref(h), ctypes.byref(cfg), 1, None, None, None, None, 0,
                              None, None, None, None) == L.LDR_EINVAL
    assert lib.ldr_views_init(None, ctypes.byref(cfg), 1, None, None, None, None, 0, None, None,
                              None, None) == L.LDR_EINVAL
    assert lib.ldr_views_update(None, None, 17, None, None, None, None) == L.LDR_EINVAL
    assert lib.ldr_draft_step(None, None, None, None, None, 0, None) == L.LDR_EINVAL
    assert lib.ldr_sample(None, 4, 10, 1.0, 0, 0, 0, None, None, None, None, 0, None) == \
        L.LDR_EINVAL
    assert lib.ldr_gumbel_fill(0, 0, 0, 0, 10, None, None) == L.LDR_EINVAL
    assert lib.ldr_gumbel_fill(0, 0, 4, 1, 10, None, None) == L.LDR_EINVAL
    fake = ctypes.c_void_p(1 << 20)   # aligned, never dereferenced: validation fails first
    ws = lib.ldr_sample_workspace_bytes(2, 64)
    for args in ((None, 2, 2, 64, fake, fake, fake, 8, L.LDR_BF16),   # no logits
                 (fake, 2, 2, 64, fake, fake, fake, 6, L.LDR_BF16),   # bf16 rank % 8
                 (fake, 2, 2, 64, fake, fake, fake, 6, L.LDR_F32),    # fp32 rank % 4
                 (fake, 2, 2, 64, fake, fake, fake, 264, L.LDR_F32),  # rank > 256
                 (fake, 2, 2, 64, fake, fake, fake, 8, 7),            # dtype
                 (fake, 0, 2, 64, fake, fake, fake, 8, L.LDR_BF16)):  # batch
        assert lib.ldr_sample_markov(*args, 1.0, 0, 0, 0, fake, fake, fake, fake, ws,
                                     None) == L.LDR_EINVAL
    vws = lib.ldr_verify_workspace_bytes(2, 3, 64)
    assert vws > 0 and lib.ldr_verify_workspace_bytes(0, 3, 64) == 0
    assert lib.ldr_verify_workspace_bytes(2, 0, 64) == 0
    for args, T, n in (((None, fake, fake, fake, 2, 3, 64), 1.0, vws),    # no target logits
                       ((fake, None, fake, fake, 2, 3, 64), 1.0, vws),    # T > 0, no draft logits
                       ((fake, fake, None, fake, 2, 3, 64), 1.0, vws),    # T > 0, no draft lse
                       ((fake, fake, fake, None, 2, 3, 64), 1.0, vws),    # no candidates
                       ((fake, fake, fake, fake, 0, 3, 64), 1.0, vws),    # batch
                       ((fake, fake, fake, fake, 2, 0, 64), 1.0, vws),    # block
                       ((fake, fake, fake, fake, 2, 3, 64), -1.0, vws),   # temperature
                       ((fake, fake, fake, fake, 2, 3, 64), float("nan"), vws),
                       ((fake, fake, fake, fake, 2, 3, 64), float("inf"), vws),
                       ((fake, fake, fake, fake, 2, 3, 64), 1.0, vws - 1)):  # short workspace
        assert lib.ldr_verify(*args, T, 0, 0, 0, fake, fake, fake, fake, n, None) == L.LDR_EINVAL
    assert lib.ldr_verify(fake, fake, fake, fake, 2, 3, 64, 1.0, -1, 0, 0, fake, fake, fake, fake,
                          vws, None) == L.LDR_EINVAL                     # negative top_k
    assert lib.ldr_views_status(None, 0, None) == L.LDR_EINVAL
    lib.ldr_views_destroy(None)
    assert lib.ldr_sample_workspace_bytes(0, 10) == 0
    assert lib.ldr_sample_workspace_bytes(256, 151936) > 0
    for code in (0, -1, -2, -3, -4, -5):
        assert lib.ldr_strerror(code)


def test_draft_step_launch_sequence():
    # fc + slot init, then per layer QKV, finishing (fp32 models; the bf16
    # attention kernel finishes q, k, v itself), attention, O, post norm,
    # gate/up, down, next norm, then the LM head
    from paper_2609_37029_amd import ldr
    for shape in (synth.TINY, synth.QWEN3_8B):
        kinds = ldr.draft_launches(shape)
        finish = ["qkv_finish"] if shape.dtype == "f32" else []
        layer = ["qkv_gemm"] + finish + ["attention", "o_gemm", "post_norm", "gate_up_gemm",
                                          "down_gemm", "next_norm"]
        assert kinds == ["fc_gemm", "slot_init"] + layer * shape.n_layers + ["lm_head"]


def test_tiled_layout_sizes_and_validation(L):
    """ldr_tiled_bytes: rows padded to 256, columns in blocks of 32 (one block
    holds all padded rows); bad
    arguments of ldr_tile_matrix are rejected on the host."""
    lib = L.lib()
    assert lib.ldr_tiled_bytes(1, 32) == 256 * 32 * 2
    assert lib.ldr_tiled_bytes(300, 96) == 512 * 96 * 2
    assert lib.ldr_tiled_bytes(151936, 4096) == 594 * 256 * 4096 * 2
    assert lib.ldr_tiled_bytes(256, 48) == 0 and lib.ldr_tiled_bytes(0, 32) == 0
    fake = ctypes.c_void_p(1 << 20)   # aligned, never dereferenced: validation fails first
    n = lib.ldr_tiled_bytes(256, 64)
    assert lib.ldr_tile_matrix(None, 256, 64, 64, fake, n, None) == L.LDR_EINVAL
    assert lib.ldr_tile_matrix(fake, 256, 48, 48, fake, n, None) == L.LDR_EINVAL     # cols % 32
    assert lib.ldr_tile_matrix(fake, 256, 64, 60, fake, n, None) == L.LDR_EINVAL     # ld < cols
    assert lib.ldr_tile_matrix(fake, 256, 64, 68, fake, n, None) == L.LDR_EINVAL     # ld % 8
    assert lib.ldr_tile_matrix(fake, 256, 64, 64, fake, n - 2, None) == L.LDR_EINVAL  # too small
    assert lib.ldr_tile_matrix(ctypes.c_void_p((1 << 20) + 8), 256, 64, 64, fake, n, None) == \
        L.LDR_EINVAL                                                                  # alignment


@pytest.mark.parametrize("drop", [0, 1, 2, 4, 3, 5, 6])
def test_view_drop_variants_state_and_launches(L, drop):
    """Ablation variants: the arena loses exactly the dropped view's bytes (the
    oracle's accounting), and without the boundary the step launches no
    boundary-fusion GEMM."""
    from oracle import views as OV
    from paper_2609_37029_amd import ldr
    for shape in (synth.TINY, synth.QWEN3_8B):
        s = shape.replace(drop_views=drop)
        assert ldr.state_bytes(s) == OV.state_bytes(s)
        kinds = ldr.draft_launches(s)
        assert ("fc_gemm" in kinds) == (not drop & 4)
        assert kinds[-1] == "lm_head"
    for flags in (8, 7):          # an unknown bit; no view at all
        bad = L.config(synth.TINY)
        bad.drop_views = flags
        assert L.lib().ldr_config_check(ctypes.byref(bad)) == L.LDR_EINVAL


def test_pooled_summary_state_and_validation(L):
    """The mean-pooled summary: arena bytes as the oracle accounts them, fixed
    in the prefix; slots must be a multiple of 32 and strides positive."""
    from oracle import views as OV
    from paper_2609_37029_amd import ldr
    for s in (synth.TINY_POOLED, synth.QWEN3_8B_POOLED,
              synth.QWEN3_8B_POOLED.replace(drop_views=1)):
        assert ldr.state_bytes(s) == OV.state_bytes(s) > 0
    for kw in (dict(pool_slots=48), dict(pool_strides=(0, 4)), dict(pool_strides=(4, -1))):
        c = L.config(synth.TINY_POOLED.replace(**kw))
        assert L.lib().ldr_config_check(ctypes.byref(c)) == L.LDR_EINVAL, kw
