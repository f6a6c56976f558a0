"""Seeded synthetic inputs for the fixed-cost drafting step.

This module only draws numbers: model shapes, weights, summary queries, target
K/V rows, boundary hidden states and anchor tokens. It holds none of the
method's arithmetic, so both the CPU oracle and the GPU path can take their
inputs from it without sharing any computation.

Shapes follow the paper's drafter (App. B.1: 5 Qwen3-style blocks, W = 256,
R = 16, views from 5 target layers) at the hidden sizes of Qwen3-8B and
Qwen3-32B, plus a small fp32 configuration that the oracle finishes in
well under a second. Distributions: matrices and embeddings ~ N(0, 0.02),
summary queries ~ N(0, 1/d) (App. B.2), target K/V rows and hidden states
~ N(0, 1), anchors uniform over the vocabulary. Every draw is seeded; a draw
on a given device is deterministic, and tests that compare devices copy the
drawn tensor instead of redrawing it.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional

import torch

# Seeds of the input streams (one independent stream per kind of input).
SEED_WEIGHTS = 0
SEED_G = 1
SEED_PREFIX = 2
SEED_ANCHOR = 3
SEED_DECODE = 4  # decode step s uses SEED_DECODE + s
SEED_GUMBEL = 5
SEED_VERIFY = 6


@dataclasses.dataclass(frozen=True)
class Shape:
    """Drafter shape. D = n_layers draft layers (one window + summary per
    layer), L_b = n_feat_layers boundary hidden states, B = block slots,
    W = window rows, R = summary queries per layer and query head."""
    name: str
    hidden: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    mlp: int
    vocab: int
    n_layers: int
    n_feat_layers: int
    block: int
    window: int
    summary: int
    rope_theta: float = 1.0e6
    ntk_alpha: float = 1.0
    rms_eps: float = 1.0e-6
    dtype: str = "bf16"  # "bf16" or "f32": weights, window rows, G, boundary h
    drop_views: int = 0  # ablation variants: 1 no window, 2 no summary, 4 no boundary (sums)
    # mean-pooled summary in place of the learned one: two banks of pool_slots
    # slots, each slot the mean K and V row of pool_strides[i] consecutive rows
    pool_strides: tuple = ()
    pool_slots: int = 0

    @property
    def qkv_out(self) -> int:
        return (self.n_q_heads + 2 * self.n_kv_heads) * self.head_dim

    @property
    def torch_dtype(self) -> torch.dtype:
        return torch.bfloat16 if self.dtype == "bf16" else torch.float32

    def replace(self, **kw) -> "Shape":
        return dataclasses.replace(self, **kw)


TINY = Shape("tiny", hidden=256, n_q_heads=4, n_kv_heads=4, head_dim=64, mlp=1024,
             vocab=4096, n_layers=1, n_feat_layers=3, block=8, window=64, summary=16,
             dtype="f32")
QWEN3_8B = Shape("qwen3-8b", hidden=4096, n_q_heads=32, n_kv_heads=8, head_dim=128,
                 mlp=12288, vocab=151936, n_layers=5, n_feat_layers=5, block=16,
                 window=256, summary=16, dtype="bf16")
# The views as the configurations word them: the last 64 rows plus mean-pooled
# summaries at strides 4 and 64 with 32 slots each (Tiny), and the same at 256
# slots per scale for the Qwen3-8B shape.
TINY_POOLED = TINY.replace(name="tiny-pooled", pool_strides=(4, 64), pool_slots=32)
QWEN3_8B_POOLED = QWEN3_8B.replace(name="qwen3-8b-pooled", pool_strides=(4, 64),
                                   pool_slots=256)
QWEN3_32B = Shape("qwen3-32b", hidden=5120, n_q_heads=64, n_kv_heads=8, head_dim=128,
                  mlp=25600, vocab=151936, n_layers=5, n_feat_layers=5, block=16,
                  window=256, summary=16, dtype="bf16")
SHAPES = {s.name: s for s in (TINY, QWEN3_8B, QWEN3_32B)}


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic workload: a shape, a batch (concurrency), a prefix length,
    a sampling temperature and, for drafting loops, the number of steps and
    the rows each step ingests."""
    name: str
    shape: Shape
    batch: int
    prefix: int
    temperature: float
    loop_steps: int = 0
    rows_per_step: int = 0


WORKLOADS = {
    w.name: w for w in (
        Workload("tiny-b1-t2048", TINY, 1, 2048, 0.0),
        Workload("qwen3-8b-b16-t32768", QWEN3_8B, 16, 32768, 1.0),
        Workload("qwen3-8b-b16-t131072-loop64", QWEN3_8B, 16, 131072, 1.0, 64, 17),
        Workload("qwen3-32b-b16-t65536", QWEN3_32B, 16, 65536, 1.0),
        Workload("tiny-pooled-b1-t2048", TINY_POOLED, 1, 2048, 0.0),
        Workload("qwen3-8b-pooled-b16-t32768", QWEN3_8B_POOLED, 16, 32768, 1.0),
    )
}
SWEEP_PREFIX = (1024, 4096, 16384, 65536, 131072, 262144)
SWEEP_BATCH = (1, 16, 64)


def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def normal(shape, std: float, seed: int, dtype=torch.float32, device="cpu") -> torch.Tensor:
    """N(0, std^2) draw, rounded once to `dtype`."""
    x = torch.randn(tuple(shape), generator=_gen(seed, device), device=device,
                    dtype=torch.float32)
    if std != 1.0:
        x.mul_(std)
    return x.to(dtype)


def _sub(seed: int, k: int) -> int:
    # Distinct, reproducible sub-seeds for the tensors of one stream.
    return (seed * 1_000_003 + k * 7919 + 12345) % (2 ** 62)


def make_weights(s: Shape, seed: int = SEED_WEIGHTS, std: float = 0.02,
                 gain_std: float = 0.0, device="cpu") -> Dict:
    """Random-init drafter weights in nn.Linear [out][in] layout.

    Norm gains are 1 + gain_std * N(0, 1) (gain_std = 0 gives the all-ones
    gains of a fresh model); every matrix and embedding is N(0, std^2).
    """
    dt = s.torch_dtype
    k = iter(range(10_000))

    def mat(*shape):
        return normal(shape, std, _sub(seed, next(k)), dt, device)

    def gain(n):
        g = normal((n,), 1.0, _sub(seed, next(k)), torch.float32, device)
        return (1.0 + gain_std * g).to(dt)

    h = s.hidden
    w = {
        "embed": mat(s.vocab, h),
        "mask_emb": mat(h),
        "pos_emb": mat(s.block, h),
        "fc_w": mat(h, s.n_feat_layers * h),
        "fc_norm": gain(h),
        "layers": [],
    }
    for _ in range(s.n_layers):
        w["layers"].append({
            "in_norm": gain(h),
            "wqkv": mat(s.qkv_out, h),
            "q_norm": gain(s.head_dim),
            "k_norm": gain(s.head_dim),
            "wo": mat(h, s.n_q_heads * s.head_dim),
            "post_norm": gain(h),
            "w_gate_up": mat(2 * s.mlp, h),
            "w_down": mat(h, s.mlp),
        })
    w["final_norm"] = gain(h)
    w["lm_head"] = mat(s.vocab, h)
    return w


def make_G(s: Shape, seed: int = SEED_G, scale: float = 1.0, device="cpu") -> torch.Tensor:
    """Summary queries G [D][Hq][R][d] ~ N(0, 1/d) (App. B.2), times `scale`
    (a sharpened G exercises the max subtraction of the log-sum-exp)."""
    std = scale / math.sqrt(s.head_dim)
    return normal((s.n_layers, s.n_q_heads, s.summary, s.head_dim), std, seed,
                  s.torch_dtype, device)


def make_rows(s: Shape, batch: int, n: int, seed: int, device="cpu", std: float = 1.0):
    """Target K and V rows [batch][n][D][Hkv][d] ~ N(0, std^2)."""
    shape = (batch, n, s.n_layers, s.n_kv_heads, s.head_dim)
    return (normal(shape, std, _sub(seed, 0), s.torch_dtype, device),
            normal(shape, std, _sub(seed, 1), s.torch_dtype, device))


def make_h(s: Shape, batch: int, seed: int, device="cpu") -> torch.Tensor:
    """Boundary hidden states [batch][L_b][hidden] ~ N(0, 1)."""
    return normal((batch, s.n_feat_layers, s.hidden), 1.0, _sub(seed, 2), s.torch_dtype,
                  device)


def make_anchors(s: Shape, batch: int, seed: int = SEED_ANCHOR, device="cpu") -> torch.Tensor:
    """Committed tokens a, uniform over [0, V), int32 [batch]."""
    return torch.randint(0, s.vocab, (batch,), generator=_gen(seed, device), device=device,
                         dtype=torch.int64).to(torch.int32)


def prefix_chunks(s: Shape, batch: int, prefix: int, chunk: int, seed: int = SEED_PREFIX,
                  device="cpu"):
    """Yield (K, V, h) chunks of a synthetic prefix of `prefix` rows per
    sequence; the last chunk is ragged. h is the boundary state after the chunk."""
    done, c = 0, 0
    while done < prefix:
        n = min(chunk, prefix - done)
        K, V = make_rows(s, batch, n, _sub(seed, 100 + c), device)
        yield K, V, make_h(s, batch, _sub(seed, 100 + c), device)
        done += n
        c += 1


def decode_rows(s: Shape, batch: int, n: int, step: int, device="cpu"):
    """K, V and h for decode step `step` (n rows per sequence)."""
    K, V = make_rows(s, batch, n, SEED_DECODE + step, device)
    return K, V, make_h(s, batch, SEED_DECODE + step, device)


def verify_round(batch: int, block: int, vocab: int, seed: int = SEED_VERIFY, device="cpu",
                 scale: float = 2.0, boost: float = 6.0, agree: float = 0.85,
                 jitter: float = 0.3):
    """A synthetic verification round: candidates y [batch][block] int32,
    draft logits z [batch][block][vocab] and target logits P
    [batch][block + 1][vocab], fp32. z ~ N(0, scale^2) plus `boost` on the
    candidate's entry; target row i is z_i plus N(0, jitter^2) noise, and with
    probability 1 - agree its boost moves from the candidate to another
    uniform token; the last target row is N(0, scale^2) with a boost on a
    uniform token."""
    g = _gen(seed, device)
    y = torch.randint(0, vocab, (batch, block), generator=g, device=device, dtype=torch.int64)
    z = torch.randn(batch, block, vocab, generator=g, device=device) * scale
    z.scatter_add_(2, y[..., None], torch.full((batch, block, 1), boost, device=device))
    P = torch.empty(batch, block + 1, vocab, device=device)
    P[:, :block] = z + torch.randn(batch, block, vocab, generator=g, device=device) * jitter
    moved = torch.rand(batch, block, generator=g, device=device) >= agree
    other = torch.randint(0, vocab, (batch, block), generator=g, device=device, dtype=torch.int64)
    shift = torch.zeros(batch, block + 1, vocab, device=device)
    shift[:, :block].scatter_add_(2, y[..., None], (-boost * moved.float())[..., None])
    shift[:, :block].scatter_add_(2, other[..., None], (boost * moved.float())[..., None])
    P[:, block] = torch.randn(batch, vocab, generator=g, device=device) * scale
    last = torch.randint(0, vocab, (batch, 1), generator=g, device=device, dtype=torch.int64)
    shift[:, block].scatter_add_(1, last, torch.full((batch, 1), boost, device=device))
    P += shift
    return y.to(torch.int32), z, P


def to_f64(t: torch.Tensor):
    """A drawn tensor as a float64 numpy array (bf16 values are exact in f64)."""
    return t.detach().to("cpu", torch.float64).numpy()


def weights_f64(w: Dict, layers: Optional[List[int]] = None) -> Dict:
    """The weight dict with every tensor as float64 numpy."""
    out = {k: to_f64(v) for k, v in w.items() if k != "layers"}
    idx = range(len(w["layers"])) if layers is None else layers
    out["layers"] = [{k: to_f64(v) for k, v in w["layers"][j].items()} for j in idx]
    return out
