"""Host-side checks of the benchmark's accounting (no GPU): the algorithmic
flops and bytes it divides by measured times, the scaling of the HBM counters
by the calibration copy, the MFMA figures from counters, and the one-GPU
contract of its command line."""
import csv
import json
import os
import subprocess
import sys

import pytest

import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def kinds_of(shape):
    from paper_2609_37029_amd import ldr
    return ldr.draft_launches(shape)


def test_step_flops_from_the_shape():
    """Flops of one Qwen3-8B batch-16 step, summed over the launch sequence,
    against the count from the parameter shapes: 2 M (weights) per layer
    GEMM (98.8 GFLOP per layer), the head's 2 M V H (318.6 GFLOP), boundary
    fusion over L_b hidden states, and 4 M H_q (B + W + R) d per attention."""
    s, batch = synth.QWEN3_8B, 16
    M, H, d = batch * s.block, s.hidden, s.head_dim
    qkv_out = (s.n_q_heads + 2 * s.n_kv_heads) * d
    layer_w = H * qkv_out + s.n_q_heads * d * H + 2 * s.mlp * H + s.mlp * H
    assert 2 * M * layer_w == 98_784_247_808
    attn = 4 * M * s.n_q_heads * (s.block + s.window + s.summary) * d
    expect = (s.n_layers * (2 * M * layer_w + attn) + 2 * M * s.vocab * H
              + 2 * batch * H * s.n_feat_layers * H)
    costs = bench.launch_costs(s, batch)
    got = sum(costs[k][1] for k in kinds_of(s))
    assert got == expect == 821_278_277_632


def test_dominant_kernel_bytes():
    """The gate/up launch the roofline uses: W_gate_up once, the normalised
    rows in, the SwiGLU output out, all bf16."""
    s, batch = synth.QWEN3_8B, 16
    M = batch * s.block
    b, f = bench.launch_costs(s, batch)["gate_up_gemm"]
    assert b == 2 * s.mlp * s.hidden * 2 + M * s.hidden * 2 + M * s.mlp * 2 == 209_715_200
    assert f == 2 * M * 2 * s.mlp * s.hidden
    # the head: W_lm once, rows in, fp32 logits out
    b, _ = bench.launch_costs(s, batch)["lm_head"]
    assert b == s.vocab * s.hidden * 2 + M * s.hidden * 2 + M * s.vocab * 4


def test_step_bytes_are_the_weights_views_and_logits():
    """Algorithmic bytes of one draft step + sampling at the Qwen3-8B shape,
    batch 16: weights 3.342 GB (layers 1.929, boundary fusion 0.168, head
    1.245), views 0.106 GB (window K/V, summary M and G) and the fp32 logits
    0.156 GB: 3.604 GB, the figure the step roofline divides by."""
    s, batch = synth.QWEN3_8B, 16
    H = s.hidden
    layers = 5 * (6144 * H + H * 4096 + 2 * 12288 * H + H * 12288) * 2
    assert layers == 1_929_379_840
    fc = H * 5 * H * 2
    head = 151936 * H * 2
    views = 5 * (16 * 2 * 8 * 256 * 128 * 2 + 16 * 32 * 16 * 128 * 4 + 32 * 16 * 128 * 2)
    logits = 16 * 16 * 151936 * 4
    got = bench.algorithmic_step_bytes(s, batch)
    assert got == layers + fc + head + views + logits
    assert abs(got / 1e9 - 3.604) < 0.002        # 3.603 GB
    # a dropped boundary has no fusion weight; a dropped window no window rows
    assert bench.algorithmic_step_bytes(s.replace(drop_views=4), batch) == got - fc
    assert bench.algorithmic_step_bytes(s.replace(drop_views=1), batch) == \
        got - 5 * 16 * 2 * 8 * 256 * 128 * 2


def _write_csv(path, rows, extra=()):
    cols = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value",
            "Start_Timestamp", "End_Timestamp"] + list(extra)
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=cols)
        w.writeheader()
        for r in rows:
            w.writerow(r)


def _dispatches(kinds, value_of, counter, t0=0, ns=1000, n_sample=2):
    """Rows of one counter: three calibration copies, a prefill update, then
    two steps (views update + commit, every draft launch, n_sample sampler
    kernels)."""
    rows, did, t = [], 0, t0

    def add(name, v):
        nonlocal did, t
        did += 1
        rows.append({"Dispatch_Id": did, "Kernel_Name": name, "Counter_Name": counter,
                     "Counter_Value": v, "Start_Timestamp": t, "End_Timestamp": t + ns})
        t += 2 * ns
    for _ in range(3):
        add("void at::native::neg_kernel_cuda(float)", value_of("neg"))
    add("void ldr::(anonymous namespace)::views_update_mfma_kernel<128, 4>(x)", 1.0)
    add("ldr::(anonymous namespace)::views_commit_kernel(int)", 1.0)
    add("void ldr::(anonymous namespace)::views_update_mfma_kernel<128, 4>(x)", 1.0)  # prefill
    for _ in range(2):
        add("void ldr::(anonymous namespace)::views_update_mfma_kernel<128, 4>(x)",
            value_of("update"))
        add("ldr::(anonymous namespace)::views_commit_kernel(int)", value_of("commit"))
        for k in kinds:
            add(f"void ldr::(anonymous namespace)::{k}_gemm_like_kernel(x)"
                if k.endswith("gemm") or k == "lm_head"
                else f"ldr::(anonymous namespace)::{k}_kernel(x)", value_of(k))
        for q in range(n_sample):
            add(f"ldr::(anonymous namespace)::sample_{q}_kernel(x)", value_of("sample"))
    return rows


@pytest.mark.parametrize("n_sample", [2, 1])
def test_traffic_scaled_by_the_calibration_copy(tmp_path, n_sample):
    """FETCH_SIZE reading half of the 1 GiB copy (factor 2) and WRITE_SIZE all
    of it (factor 1): every kind's KiB per launch times 1024 times its
    counter's factor; the views update is update + commit, the sampler its
    kernels after the head (two, or the chunk draw alone when the head forms
    the chunk log-masses), never the next step's update."""
    wl = "qwen3-8b-b16-t32768"
    kinds = kinds_of(synth.WORKLOADS[wl].shape)
    copy_kib = bench.COPY_BYTES / 1024

    def fetch(k):
        return {"neg": copy_kib / 2, "update": 30.0, "commit": 2.0, "sample": 5.0}.get(
            k, 100.0 + len(k))

    def write(k):
        return {"neg": copy_kib, "update": 7.0, "commit": 1.0, "sample": 0.5}.get(k, 10.0)
    _write_csv(tmp_path / "f.csv", _dispatches(kinds, fetch, "FETCH_SIZE", n_sample=n_sample))
    _write_csv(tmp_path / "w.csv", _dispatches(kinds, write, "WRITE_SIZE", n_sample=n_sample))
    t = bench.traffic_from_csv(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"), wl)
    assert t["calibration"]["FETCH_SIZE"]["factor"] == pytest.approx(2.0)
    assert t["calibration"]["WRITE_SIZE"]["factor"] == pytest.approx(1.0)
    g = t["kinds"]["gate_up_gemm"]
    assert g["launches"] == 2 * sum(1 for k in kinds if k == "gate_up_gemm")
    assert g["hbm_bytes_per_launch"] == pytest.approx(
        fetch("gate_up_gemm") * 1024 * 2 + write("gate_up_gemm") * 1024)
    u = t["kinds"]["views_update"]
    assert u["hbm_bytes_per_launch"] == pytest.approx((30 + 2) * 1024 * 2 + (7 + 1) * 1024)
    assert t["kinds"]["sample"]["hbm_bytes_per_launch"] == pytest.approx(
        n_sample * (5 * 1024 * 2 + 0.5 * 1024))
    assert t["sources_sha256"] == bench.source_digest()


def test_mfma_busy_from_counters(tmp_path):
    """Busy cycles summed over the 1024 SIMDs against GRBM_GUI_ACTIVE summed
    over 8 XCDs; bf16 flops = MOPS x 512; a 100 µs dispatch at 2.4 GHz."""
    wl = "qwen3-8b-b16-t32768"
    s = synth.WORKLOADS[wl].shape
    kinds = kinds_of(s)
    ns = 100_000
    active = 240_000                      # cycles of a 100 µs dispatch at 2.4 GHz
    flops = bench.launch_costs(s, 16)["gate_up_gemm"][1]
    rows = []
    for counter, val in (("SQ_VALU_MFMA_BUSY_CYCLES", 0.25 * active * 1024),
                         ("SQ_INSTS_VALU_MFMA_MOPS_BF16", flops / 512),
                         ("GRBM_GUI_ACTIVE", active * 8)):
        rows += _dispatches(kinds, lambda k, v=val: v, counter, ns=ns)
    _write_csv(tmp_path / "m.csv", rows)
    m = bench.mfma_from_csv(str(tmp_path / "m.csv"), wl)
    g = m["kinds"]["gate_up_gemm"]
    assert g["mfma_busy_frac"] == pytest.approx(0.25)
    assert g["bf16_flops_per_launch"] == pytest.approx(flops)
    assert g["gui_vs_clock"] == pytest.approx(1.0)
    assert g["tflops_under_counters"] == pytest.approx(flops / ns / 1e3)
    assert set(m["kinds"]) == {k for k in kinds if k.endswith("gemm") or k == "lm_head"}


def test_one_gpu_only_and_no_gpu_here():
    """`--gpus N` with N > 1 exits with a message; without a visible GPU the
    benchmark says so instead of measuring anything."""
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in json.loads(r.stdout.strip())["error"]
    try:
        import torch
        has_gpu = torch.cuda.is_available()
    except Exception:
        has_gpu = False
    if not has_gpu:
        r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--steps", "1"],
                           capture_output=True, text=True, timeout=300)
        assert r.returncode == 1 and "no GPU" in json.loads(r.stdout.strip())["error"]


def test_percentile():
    xs = [5.0, 1.0, 3.0, 2.0, 4.0]
    assert bench.percentile(xs, 0.5) == 3.0
    assert bench.percentile(xs, 0.0) == 1.0 and bench.percentile(xs, 1.0) == 5.0
    assert bench.percentile([], 0.5) is None


def test_step_starts_finds_each_draft_step_by_its_views_update():
    """The counter parsers find a step by its views update launch (with the
    pooling kernel, or the commit kernel of an update without rows, before the
    draft launches), skipping the prefill's updates, which are followed by
    further updates rather than the boundary-fusion GEMM."""
    names = ["neg", "views_update_mfma_kernel", "views_update_mfma_kernel",       # prefill
             "views_update_mfma_kernel", "gemm_kernel", "slot", "attn", "lse", "draw",
             "views_update_kernel", "views_pool_kernel", "gemm_kernel", "slot", "attn",
             "lse", "draw",
             "views_commit_kernel", "views_update_mfma_kernel", "views_commit_kernel",
             "gemm_kernel", "slot", "attn"]
    assert bench.step_starts(names, 3) == [(3, 4), (9, 11), (17, 19)]
    assert bench.step_starts(names[:5], 3) == []      # too few launches after it
