#!/usr/bin/env python3
"""Benchmark of the fixed-cost drafting step on one MI355X.

One step is one pass of the whole hot path for `batch` sequences: the views
ingest the 17 rows a verification pass commits (ldr_views_update), the
drafter proposes B = 16 tokens per sequence from the views alone
(ldr_draft_step), and every position is sampled (ldr_sample, temperature 1,
seeded Gumbel noise). The metric is drafted tokens per second, batch * B per
step, with every input resident in HBM before timing starts.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]
    python bench.py --sweep [--sweep-out PATH]   # latency vs prefix length and batch
    python bench.py --counters                   # short run for rocprofv3 --pmc passes
    python bench.py --traffic FETCH.csv WRITE.csv  # counters -> profiles/traffic.json

Prints one JSON line. Inputs are seeded synthetic tensors with the shapes of
the workload (random-init weights, N(0, 1) target K/V rows and hidden states).
"""
from __future__ import annotations

import argparse
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0        # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0    # MI355X dense bf16 MFMA
DEFAULT_WORKLOAD = "qwen3-8b-b16-t32768"
METRIC = "drafted tokens/sec and µs/draft step vs prefix length (Qwen3-8B shape, batch 16)"
TRAFFIC_JSON = os.path.join(ROOT, "profiles", "traffic.json")
COPY_BYTES = 1 << 30         # calibration kernel of the counter runs: reads and writes 1 GiB


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--row-major-head", action="store_true",
                    help="run the vocabulary head on the row-major lm_head (no tiled copy)")
    ap.add_argument("--markov-rank", type=int, default=0,
                    help="sample with the Markov correction (Eq. 7) of this rank instead of the "
                         "per-position sampler (0: off)")
    ap.add_argument("--temperature", type=float, default=1.0,
                    help="sampling temperature of the drafted positions (0: greedy argmax)")
    ap.add_argument("--separate-sampler", action="store_true",
                    help="draft with ldr_draft_step and sample with ldr_sample (two calls) "
                         "instead of the one call ldr_draft_step_sample")
    ap.add_argument("--no-logits", action="store_true",
                    help="greedy steps only: do not write the fp32 logits")
    ap.add_argument("--drop-views", type=int, default=0,
                    help="ablation variant: 1 no window, 2 no summary, 4 no boundary")
    ap.add_argument("--verify", action="store_true",
                    help="verify each drafted block against synthetic target logits and "
                         "commit r + 1 rows per step (closes the round on the device)")
    ap.add_argument("--cpu-seqs", type=int, default=48,
                    help="sequences in the CPU-oracle sample")
    ap.add_argument("--sweep", action="store_true")
    ap.add_argument("--sweep-out", default=os.path.join(ROOT, "sweep.json"))
    ap.add_argument("--sweep-prefix", default="1024,4096,16384,65536,131072,262144")
    ap.add_argument("--sweep-batch", default="1,16,64")
    ap.add_argument("--counters", action="store_true",
                    help="calibration copy + a few steps, to run under rocprofv3 --pmc")
    ap.add_argument("--mfma", metavar="PMC_CSV",
                    help="write profiles/mfma.json from a --pmc pass of SQ_VALU_MFMA_BUSY_CYCLES, "
                         "SQ_INSTS_VALU_MFMA_MOPS_BF16 and GRBM_GUI_ACTIVE over --counters")
    ap.add_argument("--traffic", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="turn two counter_collection.csv files into profiles/traffic.json")
    return ap.parse_args()


# ---- algorithmic bytes and flops of each launch kind --------------------------------------

def launch_costs(s, batch):
    """(bytes, flops) per launch of every draft-step kernel kind: weights read
    once, activations in, outputs out (fp32 outputs where the path keeps fp32)."""
    M = batch * s.block
    el = 2 if s.dtype == "bf16" else 4
    H, V = s.hidden, s.vocab

    def gemm(m, n, k, out_el):
        return n * k * el + m * k * el + m * n * out_el, 2 * m * n * k

    c = {
        "fc_gemm": gemm(batch, H, s.n_feat_layers * H, 4),
        "qkv_gemm": gemm(M, s.qkv_out, H, 4),
        "o_gemm": gemm(M, H, s.n_q_heads * s.head_dim, 4),
        "gate_up_gemm": (2 * s.mlp * H * el + M * H * el + M * s.mlp * el, 2 * M * 2 * s.mlp * H),
        "down_gemm": gemm(M, H, s.mlp, 4),
        "lm_head": gemm(M, V, H, 4),
    }
    # QKV finishing: fp32 projection in, q/k/v rows out, rotary table and gains
    c["qkv_finish"] = (M * s.qkv_out * (4 + el) + M * s.head_dim * 4 + 2 * s.head_dim * el, 0)
    # attention: window K/V of the layer + G and M of its heads + block q/k/v in, o out
    drop = getattr(s, "drop_views", 0)        # ablation variants read fewer sources
    pool = 0 if drop & 2 else (getattr(s, "pool_slots", 0) or 0)
    nw = (0 if drop & 1 else s.window) + 2 * pool  # window rows and pooled slot means
    nr = 0 if (drop & 2 or pool) else s.summary
    win = batch * 2 * s.n_kv_heads * nw * s.head_dim * el
    summ = s.n_q_heads * nr * s.head_dim * el + batch * s.n_q_heads * nr * s.head_dim * 4
    # bf16: the kernel also finishes q / k / v (fp32 projection rows in, the
    # rotary table and gains), and no q / k / v rows go through memory
    qkv = (M * s.qkv_out * 4 + M * s.head_dim * 4 + 2 * s.head_dim * el if el == 2
           else M * s.qkv_out * el) + M * s.n_q_heads * s.head_dim * el
    nk = s.block + nw + nr
    c["attention"] = (win + summ + qkv, 4 * M * s.n_q_heads * nk * s.head_dim)
    norm = M * H * 4 * 2 + M * H * el
    c["post_norm"] = (norm, 0)
    c["next_norm"] = (norm, 0)
    c["slot_init"] = (batch * H * 4 + M * H * (4 + el) + s.block * H * el, 0)
    return c


def algorithmic_step_bytes(s, batch):
    """Algorithmic HBM bytes of one draft step + sampling: every weight read
    once (boundary fusion, the D layers' QKV / O / gate-up / down, the
    vocabulary head), the views the attention reads (window K/V of every
    layer, the summary values M and queries G), and the fp32 logits written
    once. 3.603 GB at the Qwen3-8B shape, batch 16 (3.604 GB in round figures)."""
    el = 2 if s.dtype == "bf16" else 4
    H, d = s.hidden, s.head_dim
    drop = getattr(s, "drop_views", 0)
    pool = 0 if drop & 2 else (getattr(s, "pool_slots", 0) or 0)
    nw = (0 if drop & 1 else s.window) + 2 * pool
    nr = 0 if (drop & 2 or pool) else s.summary
    layer_w = (s.qkv_out * H + H * s.n_q_heads * d + 2 * s.mlp * H + H * s.mlp) * el
    fc_w = 0 if drop & 4 else H * s.n_feat_layers * H * el
    weights = s.n_layers * layer_w + fc_w + s.vocab * H * el
    views = s.n_layers * (batch * 2 * s.n_kv_heads * nw * d * el +
                          batch * s.n_q_heads * nr * d * 4 + s.n_q_heads * nr * d * el)
    logits = batch * s.block * s.vocab * 4
    return weights + views + logits


def update_bytes(s, batch, n):
    el = 2 if s.dtype == "bf16" else 4
    rows = batch * n * s.n_layers * s.n_kv_heads * s.head_dim * el * 2     # K/V in
    window = rows                                                        # ring write
    summ = batch * s.n_layers * s.n_q_heads * s.summary * (s.head_dim + 1) * 4 * 2  # M, eta RMW
    G = s.n_layers * s.n_q_heads * s.summary * s.head_dim * el
    h = batch * s.n_feat_layers * s.hidden * el * 2
    return rows + window + summ + G + h


# ---- setup -----------------------------------------------------------------------------

class Rig:
    """Device-resident inputs and outputs of one workload."""

    def __init__(self, torch, ldr, synth, shape, batch, prefix, chunk=4096, reuse_chunk=False,
                 tiled_head=True, markov_rank=0, verify=False, fused_head=False,
                 keep_logits=True, temperature=1.0, loop_steps=0):
        self.torch, self.ldr, self.s, self.batch = torch, ldr, shape, batch
        self.temperature = temperature
        dev = "cuda"
        self.w = synth.make_weights(shape, device=dev)
        # the vocabulary head in the library's tiled layout (a one-time copy of a frozen weight)
        self.tiled_head = tiled_head and shape.dtype == "bf16" and shape.hidden % 128 == 0
        self.dw = ldr.DraftWeights(self.w, tiled_head=self.tiled_head)
        self.G = synth.make_G(shape, device=dev)
        self.views = ldr.Views(shape, batch, self.G).init()
        if reuse_chunk:     # the same synthetic rows ingested repeatedly (timing sweeps)
            K, V, h = synth.make_rows(shape, batch, min(chunk, prefix), synth.SEED_PREFIX,
                                      device=dev) + (synth.make_h(shape, batch, synth.SEED_PREFIX,
                                                                  device=dev),)
            done = 0
            while done < prefix:
                n = min(K.shape[1], prefix - done)
                self.views.update(torch.full((batch,), n, dtype=torch.int32, device=dev), K, V, h)
                done += n
            del K, V, h
        else:
            for K, V, h in synth.prefix_chunks(shape, batch, prefix, chunk, device=dev):
                self.views.update(torch.full((batch,), K.shape[1], dtype=torch.int32,
                                             device=dev), K, V, h)
        self.n_new = shape.block + 1
        # A drafting loop (configuration 3) ingests distinct rows every step and
        # drafts from the previous step's last sampled token; other workloads
        # cycle through four decode row sets with fixed anchors.
        self.loop = loop_steps > 0
        self.rows = [synth.decode_rows(shape, batch, self.n_new, st, device=dev)
                     for st in range(loop_steps if self.loop else 4)]
        self.n = torch.full((batch,), self.n_new, dtype=torch.int32, device=dev)
        self.anchor = synth.make_anchors(shape, batch, device=dev)
        self.logits = torch.empty(batch, shape.block, shape.vocab, dtype=torch.float32,
                                  device=dev)
        self.ws = torch.empty(ldr.workspace_bytes(shape, batch), dtype=torch.uint8, device=dev)
        rows = batch * shape.block
        self.sws = torch.empty(ldr.sample_workspace_bytes(rows, shape.vocab), dtype=torch.uint8,
                               device=dev)
        self.out = (torch.empty(rows, dtype=torch.int32, device=dev),
                    torch.empty(rows, dtype=torch.float32, device=dev),
                    torch.empty(rows, dtype=torch.float32, device=dev))
        self.kinds = ldr.draft_launches(shape)
        # per-position sampling fused into the vocabulary head (ldr_draft_step_sample)
        self.fused_head = fused_head and self.tiled_head and batch * shape.block > 64
        self.keep_logits = keep_logits
        if self.fused_head:
            self.fws = torch.empty(ldr.draft_step_sample_workspace_bytes(shape, batch),
                                   dtype=torch.uint8, device=dev)
        # Markov correction (Eq. 7): seeded random correction embedding and output
        # mapping [V][rank] in the model dtype (no trained weights exist)
        self.markov_rank = markov_rank
        if markov_rank:
            g = torch.Generator(device=dev)
            g.manual_seed(synth.SEED_WEIGHTS + 17)
            self.Ec = (torch.randn(shape.vocab, markov_rank, generator=g, device=dev) *
                       0.02).to(shape.torch_dtype)
            self.Wc = (torch.randn(shape.vocab, markov_rank, generator=g, device=dev) *
                       0.02).to(shape.torch_dtype)
        # Verification (Eq. 1-2) against a synthetic target: seeded fp32 logits
        # [batch][B + 1][V] (no target model runs here). Each step then commits
        # the r + 1 rows and the emitted token that the previous step's
        # verification produced, on the device.
        self.verify = verify
        if verify:
            B = shape.block
            self.P = synth.normal((batch, B + 1, shape.vocab), 2.0, synth.SEED_VERIFY, device=dev)
            self.vws = torch.empty(ldr.verify_workspace_bytes(batch, B, shape.vocab),
                                   dtype=torch.uint8, device=dev)
            self.vout = tuple(torch.empty(batch, dtype=torch.int32, device=dev) for _ in range(3))
            self.n = self.vout[2]
            self.n.fill_(self.n_new)
            self.anchor = self.vout[1]
            self.anchor.copy_(synth.make_anchors(shape, batch, device=dev))
        torch.cuda.synchronize()
        if self.views.status() != ldr.LDR_OK:
            raise RuntimeError("views status error after prefill")

    def step(self, i, events=None):
        temperature = self.temperature
        K, V, h = self.rows[i % len(self.rows)]
        self.views.update(self.n, K, V, h)
        if self.fused_head and events is None and not self.markov_rank:
            b, B = self.batch, self.s.block
            self.ldr.draft_step_sample(self.views, self.dw, self.anchor, temperature, 5, i,
                                       logits=self.logits if self.keep_logits else None,
                                       out=tuple(t.view(b, B) for t in self.out),
                                       workspace=self.fws)
            if self.verify:
                self.verify_round(i, temperature)
            return
        if events is None:
            self.ldr.draft_step(self.views, self.dw, self.anchor, self.logits, self.ws)
        else:
            self.ldr.draft_step_events(self.views, self.dw, self.anchor, self.logits, self.ws,
                                       events)
        if self.markov_rank:
            b, B = self.batch, self.s.block
            self.ldr.sample_markov(self.logits, self.anchor, self.Ec, self.Wc, temperature, 0, 5,
                                   i, out=tuple(t.view(b, B) for t in self.out),
                                   workspace=self.sws)
        else:
            self.ldr.sample(self.logits.view(-1, self.s.vocab), temperature, 0, 5, i,
                            out=self.out, workspace=self.sws)
        if self.verify:
            self.verify_round(i, temperature)
        elif self.loop:   # the next anchor is this step's sampled y_B
            B = self.s.block
            self.anchor.copy_(self.out[0].view(self.batch, B)[:, B - 1])

    def snapshot(self):
        """Views arena, positions and anchors (restored after warm-up steps of a loop)."""
        return (self.views.arena.clone(), self.views.pos.clone(), self.anchor.clone())

    def restore(self, snap):
        self.views.arena.copy_(snap[0])
        self.views.pos.copy_(snap[1])
        self.anchor.copy_(snap[2])

    def verify_round(self, i, temperature=None):
        """ldr_verify of the step's draft; writes n (the next update's row
        counts) and the next anchors in place."""
        temperature = self.temperature if temperature is None else temperature
        b, B = self.batch, self.s.block
        self.ldr.verify(self.P, self.logits if temperature > 0 else None,
                        self.out[1].view(b, B) if temperature > 0 else None,
                        self.out[0].view(b, B), temperature, 9, i, out=self.vout,
                        workspace=self.vws)


def verify_timing(torch, rig, ev, calls=20):
    """ldr_verify alone, `calls` times between HIP events on the current
    stream: µs per call and its algorithmic bytes (the B candidate rows of the
    target read once by the lse pass; one target row and one draft row per
    sequence read by the emit pass)."""
    b, B, V = rig.batch, rig.s.block, rig.s.vocab
    stream = torch.cuda.current_stream()
    e0, e1 = ev.create(), ev.create()
    rig.verify_round(0)
    torch.cuda.synchronize()
    ev.record(e0, stream)
    for i in range(calls):
        rig.verify_round(i)
    ev.record(e1, stream)
    torch.cuda.synchronize()
    us = ev.elapsed_ms(e0, e1) * 1e3 / calls
    nbytes = b * (B + 2) * V * 4
    return {"us_per_call": us, "bytes_per_call": nbytes, "GB/s": nbytes / (us * 1e-6) / 1e9,
            "hbm_frac": nbytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBS}


BRACKET_EVERY = 1   # steps between two steps that time one launch of the bracketed kind


def time_steps(torch, rig, steps, warmup, ev=None, bracket=None):
    """Wall-clock of `steps` steps between two synchronisations; per-step
    durations from events at step boundaries; optionally events around one
    launch of the kind `bracket` in every BRACKET_EVERY-th step, taking its
    launches in turn."""
    for i in range(warmup):
        rig.step(i)
    torch.cuda.synchronize()
    marks = [ev.create() for _ in range(steps + 1)] if ev else None
    kern = None
    if ev and bracket:
        n = len(rig.kinds)
        which = [li for li, k in enumerate(rig.kinds) if k == bracket]
        kern = []
        for i in range(steps):
            evs = None
            if i % BRACKET_EVERY == 0:
                li = which[(i // BRACKET_EVERY) % len(which)]
                evs = [None] * (n + 1)
                evs[li], evs[li + 1] = ev.create(), ev.create()
            kern.append(evs)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        if marks:
            ev.record(marks[i])
        rig.step(warmup + i, events=kern[i] if kern else None)
    if marks:
        ev.record(marks[steps])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per_step = [ev.elapsed_ms(marks[i], marks[i + 1]) for i in range(steps)] if marks else []
    kernel_ms = []   # one bracketed launch per entry
    if kern:
        for evs in kern:
            if evs is None:
                continue
            li = next(j for j in range(len(rig.kinds)) if evs[j] is not None)
            kernel_ms.append(ev.elapsed_ms(evs[li], evs[li + 1]))
    return wall, per_step, kernel_ms


def kind_breakdown(torch, ldr, rig, ev, reps=5):
    """Milliseconds per step of each launch kind (events around every launch),
    after one untimed step (a kernel's first launch also loads its code)."""
    n = len(rig.kinds)
    tot = {}
    for r in range(-1, reps):
        evs = [ev.create() for _ in range(n + 1)]
        K, V, h = rig.rows[r % 4]
        rig.views.update(rig.n, K, V, h)
        ldr.draft_step_events(rig.views, rig.dw, rig.anchor, rig.logits, rig.ws, evs)
        torch.cuda.synchronize()
        if r < 0:
            continue
        for li, k in enumerate(rig.kinds):
            tot[k] = tot.get(k, 0.0) + ev.elapsed_ms(evs[li], evs[li + 1])
    return {k: v / reps for k, v in tot.items()}


def stream_bandwidth(torch, nbytes=1 << 30, reps=10):
    """Achievable HBM stream rate on this GPU: torch's elementwise copy of
    `nbytes` of fp32 (reads and writes nbytes each), median of `reps` after
    a warm-up, in GB/s of bytes moved."""
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    ts = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        dst.copy_(src)
        e1.record()
        ts.append((e0, e1))
    torch.cuda.synchronize()
    us = statistics.median(a.elapsed_time(b) * 1e3 for a, b in ts)
    del src, dst
    torch.cuda.empty_cache()
    gbs = 2 * nbytes / (us * 1e-6) / 1e9
    return {"copy_GBps": gbs, "of_peak": gbs / HBM_PEAK_GBS, "bytes_moved": 2 * nbytes,
            "kernel": "torch copy_ (fp32, 1 GiB in, 1 GiB out)"}


def percentile(xs, q):
    xs = sorted(xs)
    if not xs:
        return None
    i = min(len(xs) - 1, max(0, int(round(q * (len(xs) - 1)))))
    return xs[i]


# ---- CPU oracle baseline ----------------------------------------------------------------

def host_info():
    """Host cores and CPU model of the machine the oracle runs on."""
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except AttributeError:
        usable = os.cpu_count() or 1
    return {"nproc": usable, "cpu_count": os.cpu_count(), "cpu_model": model}


def cpu_baseline(torch, synth, rig, n_seqs):
    """The fp64 oracle on a bounded sample of the same step: views update of 17
    rows + draft forward + sampling of the B positions, for n_seqs sequences
    over views built from a 512-row prefix (the oracle's step cost does not
    depend on the prefix length once the window is full: `prefix_1k_vs_32k`
    times one sequence's step at both lengths). Also times the views update
    alone and the whole Tiny workload (prefill of 2048 rows + one step)."""
    import numpy as np
    from oracle import draft as OD
    from oracle import sample as OS
    from oracle import views as OV
    try:
        from threadpoolctl import threadpool_info
        cores = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    except Exception:
        cores = os.cpu_count() or 1
    s = rig.s
    Wt = synth.weights_f64(rig.w)
    G64 = synth.to_f64(rig.G)
    anchor = synth.make_anchors(s, n_seqs).numpy()   # seeded input, never a GPU result
    K, V, h = synth.make_rows(s, n_seqs, 512, 77) + (synth.make_h(s, n_seqs, 77),)
    Kd, Vd, hd = synth.decode_rows(s, n_seqs, s.block + 1, 0)
    states = []
    for b in range(n_seqs):
        states.append(OV.update(s, OV.empty(s), G64, synth.to_f64(K[b]), synth.to_f64(V[b]),
                                synth.to_f64(h[b])))
    upd, fwd = [], []
    t0 = time.perf_counter()
    for b in range(n_seqs):
        ta = time.perf_counter()
        st = OV.update(s, states[b], G64, synth.to_f64(Kd[b]), synth.to_f64(Vd[b]),
                       synth.to_f64(hd[b]))
        tb = time.perf_counter()
        z = OD.forward(s, Wt, st, G64, int(anchor[b]))
        OS.sample(z.astype(np.float32), rig.temperature, 0, 5, 0,
                  rows=np.arange(b * s.block, (b + 1) * s.block))
        upd.append(tb - ta)
        fwd.append(time.perf_counter() - tb)
    el = time.perf_counter() - t0

    def one_step(st, b=0):
        t = time.perf_counter()
        st2 = OV.update(s, st, G64, synth.to_f64(Kd[b]), synth.to_f64(Vd[b]),
                        synth.to_f64(hd[b]))
        z = OD.forward(s, Wt, st2, G64, int(anchor[b]))
        OS.sample(z.astype(np.float32), rig.temperature, 0, 5, 0, rows=np.arange(s.block))
        return time.perf_counter() - t

    # the step at 1K and 32K rows of prefix: one 1024-row chunk ingested repeatedly
    Kc, Vc, hc = synth.make_rows(s, 1, 1024, 78) + (synth.make_h(s, 1, 78),)
    Kc, Vc, hc = synth.to_f64(Kc[0]), synth.to_f64(Vc[0]), synth.to_f64(hc[0])
    st = OV.empty(s)
    by_prefix = {}
    for t in range(1024, 32768 + 1, 1024):
        st = OV.update(s, st, G64, Kc, Vc, hc)
        if t in (1024, 32768):
            by_prefix[str(t)] = statistics.median(one_step(st) for _ in range(3))
    del Wt
    # the whole Tiny workload: prefill 2048 rows, one update, draft, greedy sample
    tw = synth.WORKLOADS["tiny-b1-t2048"]
    ts = tw.shape
    tiny_w = synth.weights_f64(synth.make_weights(ts, device="cpu"))
    tiny_G = synth.to_f64(synth.make_G(ts, device="cpu"))
    t0 = time.perf_counter()
    tst = OV.empty(ts)
    for Kp, Vp, hp in synth.prefix_chunks(ts, 1, tw.prefix, 512, device="cpu"):
        tst = OV.update(ts, tst, tiny_G, synth.to_f64(Kp[0]), synth.to_f64(Vp[0]),
                        synth.to_f64(hp[0]))
    t1 = time.perf_counter()
    Kt, Vt, ht = synth.decode_rows(ts, 1, ts.block + 1, 0)
    tst = OV.update(ts, tst, tiny_G, synth.to_f64(Kt[0]), synth.to_f64(Vt[0]), synth.to_f64(ht[0]))
    zt = OD.forward(ts, tiny_w, tst, tiny_G, 1)
    OS.sample(zt.astype(np.float32), tw.temperature, 0, 5, 0)
    t2 = time.perf_counter()
    return {"value": n_seqs * s.block / el, "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "sample": f"{n_seqs} sequences of the workload's step: views update (17 rows) + fp64 "
                      f"draft forward + sampling of {s.block} positions over {s.vocab} tokens, "
                      f"{el:.2f} s (BLAS threads {cores}; elementwise numpy single-threaded)",
            "host": host_info(),
            "per_sequence_s": {"views_update": statistics.median(upd),
                               "draft_and_sample": statistics.median(fwd)},
            "prefix_1k_vs_32k_step_s": by_prefix,
            "tiny_b1_t2048_s": {"prefill": t1 - t0, "step": t2 - t1}}


# ---- HBM traffic from rocprofv3 counters -----------------------------------------------------

def source_digest():
    """sha256 over the library sources: counters taken on other sources are stale."""
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2609_37029_amd", "csrc")
    files = sorted(os.path.join(csrc, f) for f in os.listdir(csrc)
                   if f.endswith((".hip", ".cpp", ".h")))
    for f in files + [os.path.join(ROOT, "include", "ldr.h")]:
        h.update(os.path.basename(f).encode())
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def kernel_symbol(name):
    """Kernel name as rocprofv3 prints it, without namespaces and arguments."""
    name = name.replace("void ", "").replace("(anonymous namespace)::", "").replace("ldr::", "")
    return name.split("(")[0]


def counters_run(args, torch, ldr, synth):
    """What the --pmc passes profile: a calibration kernel of known size
    (elementwise negation of 1 GiB of fp32: reads 1 GiB, writes 1 GiB), then
    warm-up and timed steps of the workload."""
    src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        torch.neg(src, out=dst)
    torch.cuda.synchronize()
    del src, dst
    wl = synth.WORKLOADS[args.workload]
    # the benchmarked call: ldr_draft_step_sample
    rig = Rig(torch, ldr, synth, wl.shape, wl.batch, wl.prefix, fused_head=True)
    for i in range(4):
        rig.step(i)
    torch.cuda.synchronize()
    print(json.dumps({"counters_run": wl.name, "steps": 4, "kinds": rig.kinds,
                      "sources_sha256": source_digest()}), flush=True)


def step_starts(names, n_kinds):
    """(i, j) for every draft step in a dispatch sequence: the views update of
    the step starts at i (its kernels, up to the commit, end before j) and its
    n_kinds draft launches start at j with the boundary-fusion GEMM (the
    prefill's updates are followed by further updates instead)."""
    out = []
    for i, name in enumerate(names):
        if "views_update" not in name:
            continue
        j = i + 1
        while j < len(names) and ("views_pool" in names[j] or "views_commit" in names[j]):
            j += 1
        if j + n_kinds <= len(names) and "gemm" in names[j]:
            out.append((i, j))
    return out


def traffic_from_csv(fetch_csv, write_csv, workload):
    """Per-launch FETCH_SIZE / WRITE_SIZE (KiB) of every launch kind of the draft
    step, the views update and the sampler, each scaled by what the counter
    reads for the calibration kernel (COPY_BYTES in, COPY_BYTES out)."""
    import csv
    sys.path.insert(0, ROOT)
    import synth
    from paper_2609_37029_amd import ldr
    kinds = ldr.draft_launches(synth.WORKLOADS[workload].shape)

    def load(path, counter):
        disp = {}
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] != counter:
                continue
            d = disp.setdefault(int(r["Dispatch_Id"]), [r["Kernel_Name"], 0.0])
            d[1] += float(r["Counter_Value"])
        return [(k, *disp[k]) for k in sorted(disp)]

    out = {}
    for counter, path in (("FETCH_SIZE", fetch_csv), ("WRITE_SIZE", write_csv)):
        rows = load(path, counter)
        first_ldr = next(i for i, r in enumerate(rows) if "ldr::" in r[1])
        calib = [v for _, name, v in rows[:first_ldr] if "neg" in name]
        if not calib:
            raise RuntimeError(f"no calibration kernel in {path}")
        kib = statistics.median(calib)
        factor = COPY_BYTES / 1024 / kib
        per = {}
        for i, j in step_starts([r[1] for r in rows], len(kinds)):
            if j + len(kinds) + 1 > len(rows):   # the step's sampler was not recorded
                continue
            seq = rows[j:j + len(kinds)]
            per.setdefault("views_update", []).append(sum(r[2] for r in rows[i:j]))
            out.setdefault("symbols", {})["views_update"] = " + ".join(
                kernel_symbol(r[1]) for r in rows[i:j])
            for k, (_, kname, v) in zip(kinds, seq):
                e = per.setdefault(k, [])
                e.append(v)
                out.setdefault("symbols", {})[k] = kernel_symbol(kname)
            # the sampler's kernels after the head (the chunk draw alone when
            # the head forms the chunk log-masses), up to the next views update
            tail = []
            for r in rows[j + len(kinds):j + 2 + len(kinds)]:
                if "views_" in r[1]:
                    break
                tail.append(r)
            per.setdefault("sample", []).append(sum(v for _, _, v in tail))
            out.setdefault("symbols", {})["sample"] = " + ".join(kernel_symbol(r[1]) for r in tail)
        out.setdefault("calibration", {})[counter] = {"kib_read_by_counter": kib,
                                                     "factor": factor}
        for k, vs in per.items():
            e = out.setdefault("kinds", {}).setdefault(k, {})
            e[counter + "_kib_per_launch"] = statistics.mean(vs)
            e["launches"] = len(vs)
            e[counter.split("_")[0].lower() + "_bytes_per_launch"] = \
                statistics.mean(vs) * 1024 * factor
    for e in out["kinds"].values():
        e["hbm_bytes_per_launch"] = e.get("fetch_bytes_per_launch", 0) + \
            e.get("write_bytes_per_launch", 0)
    out["workload"] = workload
    out["sources_sha256"] = source_digest()
    return out


def mfma_from_csv(path, workload):
    """Per-launch MFMA figures of the GEMM launch kinds from one rocprofv3 --pmc
    pass over `bench.py --counters` with SQ_VALU_MFMA_BUSY_CYCLES,
    SQ_INSTS_VALU_MFMA_MOPS_BF16 and GRBM_GUI_ACTIVE: the MFMA busy fraction
    (busy cycles summed over the SIMDs / (GPU active cycles x SIMDs)), the bf16
    flops the instructions did (MOPS x 512) and the dispatch duration. The CSV
    holds one GRBM_GUI_ACTIVE value per dispatch summed over the 8 XCDs' GRBM
    blocks, so the GPU's active cycles are that value / 8; `gui_vs_clock`
    compares them with the dispatch duration at 2.4 GHz."""
    import csv
    sys.path.insert(0, ROOT)
    import synth
    from paper_2609_37029_amd import ldr
    kinds = ldr.draft_launches(synth.WORKLOADS[workload].shape)
    disp = {}
    for r in csv.DictReader(open(path)):
        d = disp.setdefault(int(r["Dispatch_Id"]), {"name": r["Kernel_Name"], "busy": 0.0,
                                                    "mops": 0.0, "gui": 0.0,
                                                    "ns": int(r["End_Timestamp"]) -
                                                          int(r["Start_Timestamp"])})
        v = float(r["Counter_Value"])
        if r["Counter_Name"] == "SQ_VALU_MFMA_BUSY_CYCLES":
            d["busy"] += v
        elif r["Counter_Name"] == "SQ_INSTS_VALU_MFMA_MOPS_BF16":
            d["mops"] += v
        elif r["Counter_Name"] == "GRBM_GUI_ACTIVE":
            d["gui"] = max(d["gui"], v)
    rows = [disp[k] for k in sorted(disp)]
    simds, xcds, ghz = 256 * 4, 8, 2.4
    per = {}
    for _, j in step_starts([r["name"] for r in rows], len(kinds)):
        seq = rows[j:j + len(kinds)]
        for k, d in zip(kinds, seq):
            if k.endswith("gemm") or k == "lm_head":
                per.setdefault(k, []).append(d)
    out = {"workload": workload, "sources_sha256": source_digest(), "simds": simds, "kinds": {}}
    for k, ds in per.items():
        busy = statistics.mean(d["busy"] / (d["gui"] / xcds * simds) for d in ds if d["gui"] > 0)
        flops = statistics.mean(d["mops"] * 512 for d in ds)
        ns = statistics.mean(d["ns"] for d in ds)
        gui = statistics.mean(d["gui"] / xcds for d in ds)
        out["kinds"][k] = {"symbol": kernel_symbol(ds[0]["name"]), "launches": len(ds),
                           "mfma_busy_frac": busy, "bf16_flops_per_launch": flops,
                           "us_per_launch_under_counters": ns / 1e3,
                           "tflops_under_counters": flops / ns / 1e3,
                           "frac_of_bf16_peak": flops / ns / 1e3 / BF16_PEAK_TFLOPS,
                           "gui_vs_clock": gui / (ns * ghz)}
    return out


def traffic_for(kind):
    """HBM bytes per launch of `kind` from profiles/traffic.json, or None when
    absent or taken on other library sources."""
    try:
        with open(TRAFFIC_JSON) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("sources_sha256") != source_digest():
        return None
    e = t.get("kinds", {}).get(kind)
    return e.get("hbm_bytes_per_launch") if e else None


def gemm_mfma_from_counters(s, batch, kinds):
    """bf16 flops of all GEMMs of one step over their summed dispatch time,
    from profiles/mfma.json (rocprofv3 counter pass), or None when it is
    absent or was taken on other library sources."""
    try:
        with open(os.path.join(ROOT, "profiles", "mfma.json")) as f:
            m = json.load(f)
    except (OSError, ValueError):
        return None
    if m.get("sources_sha256") != source_digest():
        return None
    flops = us = 0.0
    for k, e in m.get("kinds", {}).items():
        n = sum(1 for x in kinds if x == k)
        flops += e["bf16_flops_per_launch"] * n
        us += e["us_per_launch_under_counters"] * n
    if us <= 0:
        return None
    tf = flops / (us * 1e-6) / 1e12
    return {"tflops": tf, "frac": tf / BF16_PEAK_TFLOPS, "source": "profiles/mfma.json"}


# ---- main --------------------------------------------------------------------------------

def main():
    args = parse()
    if args.mfma:
        m = mfma_from_csv(args.mfma, args.workload)
        with open(os.path.join(ROOT, "profiles", "mfma.json"), "w") as f:
            json.dump(m, f, indent=1)
        print(json.dumps({k: round(v["mfma_busy_frac"], 3) for k, v in m["kinds"].items()}))
        return
    if args.traffic:
        t = traffic_from_csv(args.traffic[0], args.traffic[1], args.workload)
        os.makedirs(os.path.dirname(TRAFFIC_JSON), exist_ok=True)
        with open(TRAFFIC_JSON, "w") as f:
            json.dump(t, f, indent=1)
        print(json.dumps({k: round(v["hbm_bytes_per_launch"] / 1e6, 2)
                          for k, v in t["kinds"].items()}))
        return
    if args.gpus != 1:
        print(json.dumps({"error": f"--gpus {args.gpus}: this benchmark runs on one GPU only; "
                                   "the drafting step shards by sequence with no exchange, so "
                                   "N GPUs run N independent copies"}))
        sys.exit(2)
    import torch

    import synth
    from paper_2609_37029_amd import ldr
    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}))
        sys.exit(1)
    torch.cuda.set_device(0)
    if args.sweep:
        return sweep(args, torch, ldr, synth)
    if args.counters:
        return counters_run(args, torch, ldr, synth)

    wl = synth.WORKLOADS[args.workload]
    s, batch = wl.shape, wl.batch
    if args.drop_views:
        s = s.replace(drop_views=args.drop_views)
    loop = wl.loop_steps if not (args.verify or args.markov_rank) else 0
    if loop:
        args.steps = loop       # the loop's own length: every step is timed
    rig = Rig(torch, ldr, synth, s, batch, wl.prefix, tiled_head=not args.row_major_head,
              markov_rank=args.markov_rank, verify=args.verify,
              fused_head=not args.separate_sampler,
              keep_logits=not args.no_logits, temperature=args.temperature, loop_steps=loop)
    ev = ldr.HipEvents()
    costs = launch_costs(s, batch)
    # which launch kind dominates the step (events around every launch, outside the timed run)
    snap = rig.snapshot() if loop else None
    br = kind_breakdown(torch, ldr, rig, ev)
    dom = max(br, key=lambda k: br[k])
    if loop:   # warm-up steps on the same state, then back to the loop's start
        for i in range(args.warmup):
            rig.step(i)
        torch.cuda.synchronize()
        rig.restore(snap)
        args_warmup_run = 0
    else:
        args_warmup_run = args.warmup
    if rig.fused_head:
        # ldr_draft_step_sample records no per-launch events: the timed run has
        # events at step boundaries only, and the dominant kernel (a draft-layer
        # launch, the same kernel on both paths) is timed over as many steps of
        # the bracketed separate path right after it
        wall, per_step, _ = time_steps(torch, rig, args.steps, args_warmup_run, ev=ev)
        t_final = int(rig.views.pos.min().item())   # the timed steps' prefix, before the bracketed run
        rig.fused_head = False
        _, _, kern = time_steps(torch, rig, args.steps, 0, ev=ev, bracket=dom)
        rig.fused_head = True
    else:
        wall, per_step, kern = time_steps(torch, rig, args.steps, args_warmup_run, ev=ev,
                                          bracket=dom)
        t_final = int(rig.views.pos.min().item())
    torch.cuda.synchronize()
    ms = wall / args.steps * 1e3
    tokens = batch * s.block * args.steps
    launches_of_dom = sum(1 for k in rig.kinds if k == dom)
    dom_ms = statistics.mean(kern)
    dom_bytes = costs[dom][0]
    achieved = dom_bytes / (dom_ms * 1e-3) / 1e9
    step_bytes = algorithmic_step_bytes(s, batch)
    upd_bytes = update_bytes(s, batch, s.block + 1)
    step_flops = sum(costs[k][1] for k in rig.kinds)
    out = {
        "metric": METRIC, "value": tokens / wall, "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": s.dtype,
        "data": "synthetic (seeded random-init weights, N(0,1) target K/V rows and hidden "
                "states; prefix rows ingested through ldr_views_update before timing)",
        "config": {"workload": wl.name, "shape": s.name, "batch": batch, "block": s.block,
                   "prefix": wl.prefix, "rows_per_update": s.block + 1,
                   "temperature": rig.temperature,
                   "window": s.window, "summary": s.summary, "draft_layers": s.n_layers,
                   "lm_head_layout": "tiled" if rig.tiled_head else "row-major",
                   "sampler": (f"markov rank {rig.markov_rank}" if rig.markov_rank else
                               ("ldr_draft_step_sample: " +
                                ("argmax in the vocabulary head's epilogue" +
                                 ("" if rig.keep_logits else ", logits not written")
                                 if rig.temperature == 0 else
                                 "chunk log-masses in the vocabulary head's epilogue, "
                                 "then the chunk draw"))
                               if rig.fused_head else "ldr_draft_step + ldr_sample"),
                   "views": {0: "window + summary + boundary", 1: "no window", 2: "no summary",
                             4: "no boundary"}.get(s.drop_views, f"drop {s.drop_views}")},
        "us_per_step": {"p10": percentile(per_step, .1) * 1e3, "p50": percentile(per_step, .5) * 1e3,
                        "p90": percentile(per_step, .9) * 1e3},
        "roofline": {"bound": "hbm", "kernel": dom, "achieved": achieved, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS, "traffic": traffic_for(dom),
                     "bytes_per_launch": dom_bytes, "us_per_launch": dom_ms * 1e3,
                     "launches_per_step": launches_of_dom, "launches_timed": len(kern)},
        "step_roofline": {"algorithmic_bytes": step_bytes, "update_bytes": upd_bytes,
                          "flops": step_flops,
                          "hbm_frac": (step_bytes + upd_bytes) / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
                          "gemm_mfma": gemm_mfma_from_counters(s, batch, rig.kinds)},
        "state_bytes_per_seq": ldr.state_bytes(s),
    }
    if loop:
        out["config"]["loop_steps"] = loop
        out["config"]["anchor"] = "the previous step's sampled y_B"
        out["config"]["prefix_after_loop"] = t_final
        out["us_per_step"]["first"] = per_step[0] * 1e3
        out["us_per_step"]["last"] = per_step[-1] * 1e3
    out["stream_bw"] = stream_bandwidth(torch)
    if rig.verify:
        out["config"]["rows_per_update"] = "r + 1 from ldr_verify"
        out["verify"] = verify_timing(torch, rig, ev)
    ev.close()
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(torch, synth, rig, args.cpu_seqs)
    print(json.dumps(out), flush=True)


def sweep(args, torch, ldr, synth):
    s = synth.QWEN3_8B
    ev = ldr.HipEvents()
    res = []
    for batch in [int(x) for x in args.sweep_batch.split(",")]:
        for prefix in [int(x) for x in args.sweep_prefix.split(",")]:
            rig = Rig(torch, ldr, synth, s, batch, prefix, reuse_chunk=True,
                      tiled_head=not args.row_major_head, fused_head=not args.separate_sampler)
            wall, per_step, _ = time_steps(torch, rig, args.steps, args.warmup, ev=ev)
            r = {"batch": batch, "prefix": prefix, "us_p50": percentile(per_step, .5) * 1e3,
                 "us_p10": percentile(per_step, .1) * 1e3,
                 "us_p90": percentile(per_step, .9) * 1e3,
                 "tokens_per_s": batch * s.block * args.steps / wall,
                 "state_bytes_per_seq": ldr.state_bytes(s)}
            res.append(r)
            print(json.dumps(r), file=sys.stderr, flush=True)
            del rig
            torch.cuda.empty_cache()
    flat = {}
    for batch in sorted({r["batch"] for r in res}):
        xs = [r["us_p50"] for r in res if r["batch"] == batch]
        flat[str(batch)] = (max(xs) - min(xs)) / min(xs)
    os.makedirs(os.path.dirname(os.path.abspath(args.sweep_out)), exist_ok=True)
    with open(args.sweep_out, "w") as f:
        json.dump({"shape": s.name, "points": res, "variation": flat}, f, indent=1)
    print(json.dumps({"metric": "draft-step latency vs prefix length", "shape": s.name,
                      "variation_max_over_min_minus_1": flat, "points": len(res),
                      "out": args.sweep_out}), flush=True)


if __name__ == "__main__":
    main()
