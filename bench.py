#!/usr/bin/env python3
"""Benchmark of one host's share of APB prefill attention on one MI355X.

One step = the whole host-share hot path on one batch of synthetic input:
``apb_compress_select`` (top-l_p of the local block's scores + gather into
slot host_idx of the rank-major passing buffer) and ``apb_attention_fwd``
(modified-mask attention reading the earlier hosts' slots in place).  The
compressor's output is not read by the same host's attention; they run back
to back on one stream (``--overlap``: concurrently on two).  Inputs are
resident in HBM before timing starts.

Prints ONE JSON line.  ``value`` is unmasked attention TFLOP/s over the
whole step; ``roofline`` reports the attention kernel alone (HIP events on
the launch stream); ``cpu_baseline`` is the fp64 oracle timed on a bounded
sample on the host cores.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0  # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0
KERNEL_SOURCES = ["paper_2502_12085_amd/csrc/apb_attention.hip"]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "attention_llama8b_128k_traffic.json")


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(workload: str):
    """HBM bytes per attention launch from the committed rocprofv3 counter
    runs, if they were taken on the current kernel source and workload."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("kernel_source_hash") != kernel_source_hash() or t.get("workload") != workload:
        return None
    return t.get("hbm_bytes_per_launch")


def _oracle_threads() -> int:
    """Threads the oracle's BLAS calls use on this host."""
    try:
        from threadpoolctl import threadpool_info
        return int(max([i.get("num_threads", 1) for i in threadpool_info()] or [1]))
    except Exception:  # noqa: BLE001
        return os.cpu_count() or 1


def host_info() -> dict:
    """The host the oracle runs on: CPU model and the cores this process may
    use (the container's share, not the machine's)."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        nproc = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        nproc = os.cpu_count() or 1
    return {"cpu_model": model, "nproc": nproc}


def cpu_baseline(wl, inp, budget_s: float):
    """fp64 oracle on a bounded sample: whole query heads (all rows), as many
    as fit the time budget (at least one)."""
    import numpy as np
    import oracle
    cores = _oracle_threads()
    p = wl.problem
    flops_head = oracle.attention_flops(1, p.head_dim, p.anchor_len, p.local_len, p.passing_rows)
    t0 = time.perf_counter()
    heads = 0
    while True:
        oracle.attention_ref(inp["q"], inp["k"], inp["v"], inp["k_pass"], inp["v_pass"],
                             anchor_len=p.anchor_len, heads=np.array([heads]))
        heads += 1
        el = time.perf_counter() - t0
        if el > budget_s or heads >= p.n_q_heads or el / heads * (heads + 1) > 1.5 * budget_s:
            break
    el = time.perf_counter() - t0
    return {"value": round(flops_head * heads / el / 1e12, 6), "unit": "TFLOP/s",
            "cores": int(cores), "kind": "oracle",
            "sample": f"{heads} of {p.n_q_heads} query heads, all {p.rows} rows, fp64 NumPy; "
                      f"{el:.1f} s wall",
            "seconds": round(el, 3), **host_info()}


def busy_ahead(stream, ms: float = 20.0) -> None:
    """Occupy the GPU with a spin kernel on `stream` while the host enqueues
    the timed launches behind it, so that launches of a few microseconds run
    back to back and their events do not include host submission gaps."""
    import torch
    torch.cuda.set_stream(stream)
    torch.cuda._sleep(int(ms * 1e-3 * 2.4e9))


def warm_up(step, min_steps: int, seconds: float = 0.2) -> float:
    """Run `step` (one synchronised call each) until at least `min_steps`
    calls and `seconds` of them have passed, and return the last call's
    milliseconds: from idle the shader clock takes some tens of milliseconds
    of load to settle (measured: 30 ms of back-to-back 32K attention launches
    ran up to 20% slower than the ones after), so a few short warm-up steps
    would leave the timed ones on the way up."""
    import torch
    t0 = time.perf_counter()
    n, last = 0, 0.0
    while n < min_steps or time.perf_counter() - t0 < seconds:
        t1 = time.perf_counter()
        step()
        torch.cuda.synchronize()
        last = (time.perf_counter() - t1) * 1e3
        n += 1
    return last


def parse_smi_metric(text: str):
    """Socket watts and the per-XCD shader clocks (MHz) from the text of
    `amd-smi metric -p -c` for one GPU: (None, []) where it prints neither."""
    import re
    m = re.search(r"SOCKET_POWER:\s*([0-9.]+)\s*W", text)
    clks, section = [], ""
    for line in text.splitlines():
        h = re.match(r"\s*([A-Z]+_[0-9]+):\s*$", line)
        if h:
            section = h.group(1)
            continue
        c = re.match(r"\s*CLK:\s*([0-9]+)\s*MHz", line)
        if c and section.startswith("GFX_"):
            clks.append(int(c.group(1)))
    return (float(m.group(1)) if m else None), clks


def parse_power_cap(text: str):
    """The package power cap (W) from `rocm-smi --showmaxpower`, or None."""
    import re
    m = re.search(r"Max Graphics Package Power \(W\):\s*([0-9.]+)", text)
    return float(m.group(1)) if m else None


def sample_power(launch, seconds: float = 3.0) -> dict:
    """Socket power and shader clock while `launch` (one attention call) runs
    back to back: about `seconds` of launches are queued and the vendor's SMI
    tool is read every quarter second while they run.  `samples` holds each
    reading (seconds since the queue started, socket watts, mean XCD clock in
    MHz); `socket_power_w` and `gfx_clk_mhz` (one per XCD) come from the
    readings taken after the first second, while the chip was still busy
    (the power manager ramps the clock up from idle over a fraction of a
    second).  Context for the roofline fraction: the chip's clock under a
    matrix load is set by its power cap.  Values are None where the tool is
    missing or prints something else."""
    import shutil
    import statistics
    import subprocess
    import torch

    def run(cmd):
        try:
            return subprocess.run(cmd, capture_output=True, text=True, timeout=20).stdout
        except (OSError, subprocess.SubprocessError):
            return ""

    out = {"during": "back-to-back launches of the attention kernel above",
           "socket_power_w": None, "power_cap_w": None, "gfx_clk_mhz": None, "samples": []}
    smi = shutil.which("amd-smi") or "/opt/rocm/bin/amd-smi"
    rsmi = shutil.which("rocm-smi") or "/opt/rocm/bin/rocm-smi"
    if not os.path.exists(smi):
        return out
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    launch()
    e1.record()
    torch.cuda.synchronize()
    n = max(1, int(seconds / max(e0.elapsed_time(e1) * 1e-3, 1e-4)))
    done = torch.cuda.Event()
    t0 = time.perf_counter()
    for _ in range(n):
        launch()
    done.record()
    steady = []
    while True:
        time.sleep(0.25)
        watts, clks = parse_smi_metric(run([smi, "metric", "-p", "-c"]))
        t = time.perf_counter() - t0
        busy = not done.query()
        if not busy:
            break
        mean_clk = round(sum(clks) / len(clks)) if clks else None
        out["samples"].append([round(t, 2), watts, mean_clk])
        if t >= 1.0 and watts is not None:
            steady.append((watts, clks))
    torch.cuda.synchronize()
    if steady:
        out["socket_power_w"] = statistics.median(w for w, _ in steady)
        out["gfx_clk_mhz"] = steady[-1][1] or None
    cap = run([rsmi, "--showmaxpower"]) if os.path.exists(rsmi) else ""
    out["power_cap_w"] = parse_power_cap(cap)
    out["launches"] = n
    out["tools"] = "amd-smi metric -p -c; rocm-smi --showmaxpower"
    return out


def bench_mfma_ceiling(steps: int, seed: int = 0) -> dict:
    """Matrix-core ceiling on this chip: the probe library's back-to-back
    32x32x16 bf16 MFMA loop on random N(0,1) operands (one workgroup of 8
    waves per CU, four independent accumulators per wave, no other work),
    median of `steps` launches of about 2.5 ms each.  Under this load the
    shader clock settles well below its 2.4 GHz peak, so the rate is the
    ceiling a bf16 kernel can reach here, below the nominal peak."""
    import torch
    from paper_2502_12085_amd import probe

    n_wg, iters = 256, 16384  # exactly one workgroup per CU, one round
    g = torch.Generator(device="cpu").manual_seed(seed)
    ops = torch.randn(8192, generator=g).to(torch.bfloat16).cuda()
    sink = torch.empty(n_wg * 512, dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    for _ in range(2):
        probe.mfma_bf16(ops, sink, n_wg, iters, stream)
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(steps)]
    for e0, e1 in ev:
        e0.record(stream)
        probe.mfma_bf16(ops, sink, n_wg, iters, stream)
        e1.record(stream)
    torch.cuda.synchronize()
    ms = sorted(a.elapsed_time(b) for a, b in ev)[len(ev) // 2]
    tf = probe.mfma_flops(n_wg, iters) / (ms * 1e-3) / 1e12
    return {"tflops": round(tf, 1), "frac_of_nominal_peak": round(tf / PEAK_BF16_TFLOPS, 4),
            "kernel": "mfma_loop_kernel (libapb_probe.so)",
            "operands": "random N(0,1) bf16", "workgroups": n_wg, "waves_per_cu": 8,
            "ms": round(ms, 3), "timing": f"median of {steps} launches, HIP events"}


def bench_layer(lw, steps: int, warmup: int, seed: int = 0) -> dict:
    """One host's whole layer (Alg. 2 with the model's layer around the host
    share): apb_layer_fwd on synthetic weights, inputs resident in HBM, HIP
    events around each call on the launch stream."""
    import numpy as np
    import torch
    from paper_2502_12085_amd import apb, inputs

    p = lw.problem
    inp = inputs.make_layer_inputs(lw, seed)

    def dev(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()

    w = {k: dev(inp["w"][v]) for k, v in (("ln1", "ln1"), ("w_qkv", "w_qkv"), ("w_o", "w_o"),
                                         ("ln2", "ln2"), ("w_gate", "w_gate"), ("w_up", "w_up"),
                                         ("w_down", "w_down"), ("r_w1", "w1"))}
    for k, v in (("r_b1", "b1"), ("r_w2", "w2"), ("r_b2", "b2")):
        w[k] = torch.from_numpy(np.ascontiguousarray(inp["w"][v])).cuda()
    hidden, pos = dev(inp["hidden"]), torch.from_numpy(inp["pos"]).cuda()
    pk = torch.zeros((p.n_hosts, p.n_kv_heads, p.pass_len, p.head_dim), dtype=torch.bfloat16,
                     device="cuda")
    pv = torch.zeros_like(pk)
    pk[:p.host_idx] = dev(inp["k_pass"])
    pv[:p.host_idx] = dev(inp["v_pass"])
    kc = torch.empty((p.n_kv_heads, p.rows, p.head_dim), dtype=torch.bfloat16, device="cuda")
    vc = torch.empty_like(kc)
    out = torch.empty((p.rows, lw.hidden), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(apb.layer_workspace_size(lw), dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()

    def call():
        apb.layer_fwd(lw, w, hidden, pos, kc, vc, pk, pv, out, ws, stream)

    warm_up(call, warmup)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(steps)]
    for e0, e1 in ev:
        e0.record(stream)
        call()
        e1.record(stream)
    torch.cuda.synchronize()
    ms = sorted(a.elapsed_time(b) for a, b in ev)[len(ev) // 2]
    flops = apb.layer_flops(lw)
    return {"workload": lw.name, "hidden": lw.hidden, "intermediate": lw.intermediate,
            "rows": p.rows, "ms": round(ms, 3), "flops": flops,
            "tflops": round(flops / (ms * 1e-3) / 1e12, 1),
            "frac_of_peak": round(flops / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
            "kernels": "rmsnorm, gemm(QKV), rope, scorer, compressor, attention, gemm(O), "
                       "rmsnorm, gemm(gate/up + SwiGLU), gemm(down)",
            "timing": f"median of {steps} calls, HIP events", "weights": "synthetic",
            "paper_context": {"a800_block_ms": 80.18,
                              "note": "8xA800 per-block wall time at 128K (the paper's "
                                      "block breakdown); another machine"}}


def bench_stage2(wl, steps: int, warmup: int, seed: int = 0, cpu_budget: float = 0.0) -> dict:
    """Decoding stage (Alg. 3) at the same layer shape: the last host's
    partial attention over its cache plus the new tokens' K/V, and MergeScore
    of the H hosts' partials (the other hosts' partials are synthetic).  HIP
    events on the launch stream; inputs resident in HBM."""
    import numpy as np
    import torch
    from paper_2502_12085_amd import apb, inputs

    case = inputs.make_decode_inputs(wl, seed, hosts=1)
    kc, vc = case["caches"][0]

    def dev(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()

    q, dkc, dvc, kn, vn = dev(case["q"]), dev(kc), dev(vc), dev(case["k_new"]), dev(case["v_new"])
    n_q, n_kv, d, n_new, lc, H = (wl.n_q_heads, wl.n_kv_heads, wl.head_dim, wl.n_new,
                                  wl.cache_len, wl.n_hosts)
    rows = n_q * n_new
    prob = apb.DecodeProblem(n_q, n_kv, d, lc, n_new, 1)
    ws = torch.empty(apb.decode_workspace_size(prob), dtype=torch.uint8, device="cuda")
    g = torch.Generator(device="cuda").manual_seed(seed)
    parts_o = torch.randn((H, rows, d), generator=g, device="cuda", dtype=torch.float32)
    parts_l = torch.randn((H, rows), generator=g, device="cuda", dtype=torch.float32)
    o = torch.empty((rows, d), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((rows,), dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()

    def step(events=None):
        if events:
            events[0].record(stream)
        apb.decode_attention(prob, q, dkc, dvc, kn, vn, parts_o[H - 1].view(n_q, n_new, d),
                             parts_l[H - 1].view(n_q, n_new), ws, 0.0, stream)
        if events:
            events[1].record(stream)
        apb.merge_partials(parts_o, parts_l, o, lse, stream)
        if events:
            events[2].record(stream)

    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
    warm_up(step, warmup)
    busy_ahead(stream)
    for e in ev:
        step(e)
    torch.cuda.synchronize()
    t_dec = [a.elapsed_time(b) for a, b, _ in ev]
    t_mrg = [b.elapsed_time(c) for _, b, c in ev]
    dec_us = 1e3 * sorted(t_dec)[len(t_dec) // 2]
    mrg_us = 1e3 * sorted(t_mrg)[len(t_mrg) // 2]
    keys = lc + n_new
    dec_bytes = 2 * rows * d + 2 * 2 * n_kv * keys * d + 4 * rows * d + 4 * rows
    mrg_bytes = H * rows * (d + 1) * 4 + rows * d * 2 + rows * 4
    # 4d flops per visible (row, key) pair: on the last host new token j sees
    # the cache and new tokens 0..j
    pairs = n_new * lc + n_new * (n_new + 1) // 2
    dec_flops = 4.0 * d * n_q * pairs
    cpu = None
    if cpu_budget > 0:
        import oracle
        t0 = time.perf_counter()
        reps = 0
        while True:
            oracle.decode_attention_ref(case["q"], kc, vc, case["k_new"], case["v_new"])
            reps += 1
            if time.perf_counter() - t0 > cpu_budget or reps >= 20:
                break
        el = (time.perf_counter() - t0) / reps
        cpu = {"value": round(dec_bytes / el / 1e9, 3), "unit": "GB/s", "us": round(el * 1e6, 1),
               "cores": _oracle_threads(), "kind": "oracle",
               "sample": f"the whole partial attention (fp64 NumPy), {reps} run(s)"}
    return {"workload": wl.name, "n_hosts": H, "cache_len": lc, "n_new": n_new,
            "n_q_heads": n_q, "n_kv_heads": n_kv, "head_dim": d,
            "decode_us": round(dec_us, 2), "decode_algorithmic_bytes": dec_bytes,
            "decode_gbs": round(dec_bytes / (dec_us * 1e-6) / 1e9, 1),
            "decode_hbm_frac": round(dec_bytes / (dec_us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4),
            "decode_flops": dec_flops,
            "decode_mfma_frac": round(dec_flops / (dec_us * 1e-6) / 1e12 / PEAK_BF16_TFLOPS, 4),
            "arithmetic_intensity": round(dec_flops / dec_bytes, 1),
            "merge_us": round(mrg_us, 2), "merge_algorithmic_bytes": mrg_bytes,
            # the library's plan: eight-wave ping-pong workgroups once a GQA
            # group has four 32-row blocks, one-wave workgroups below that
            "kernel": ("decode_pingpong_kernel" if (n_q // n_kv) * n_new >= 128 else "decode_partial_kernel")
            + f"<{d}> + merge_kernel",
            "bound": "hbm", "timing": f"median of {steps} back-to-back launches, HIP events",
            "cpu_baseline": cpu}


def bench_scorer(wl, steps: int, warmup: int, seed: int = 0, cpu_budget: float = 0.0) -> dict:
    """Retaining-head scorer (Sec. 3.4, App. B) on the same host share with
    synthetic weights: bf16 GEMM [Lb x (n_q+2n_kv)d] x [. x 1024] fused with
    SiLU and the per-KV-head output layer.  HIP events on the launch stream."""
    import numpy as np
    import torch
    from paper_2502_12085_amd import apb, inputs

    p = wl.problem
    inp = inputs.make_inputs(wl, seed)
    w = inputs.make_scorer_weights(p.n_q_heads, p.n_kv_heads, p.head_dim, seed=seed)

    def dev(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()

    def f32(a):
        return torch.from_numpy(np.ascontiguousarray(a)).cuda()

    q, k, v, w1 = dev(inp["q"]), dev(inp["k"]), dev(inp["v"]), dev(w["w1"])
    b1, w2, b2 = f32(w["b1"]), f32(w["w2"]), f32(w["b2"])
    hidden = inputs.SCORER_HIDDEN
    sp = apb.ScorerProblem(p.anchor_len, p.local_len, p.n_q_heads, p.n_kv_heads, p.head_dim, hidden)
    ws = torch.empty(apb.scorer_workspace_size(sp), dtype=torch.uint8, device="cuda")
    scores = torch.empty((p.n_kv_heads, p.local_len), dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    warm_up(lambda: apb.retaining_scores(sp, q, k, v, w1, b1, w2, b2, scores, ws, stream), warmup)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(steps)]
    # no spin ahead: a call is long beside its submission, and a spin would
    # let the clock rise above what back-to-back calls hold
    for e0, e1 in ev:
        e0.record(stream)
        apb.retaining_scores(sp, q, k, v, w1, b1, w2, b2, scores, ws, stream)
        e1.record(stream)
    torch.cuda.synchronize()
    t = [a.elapsed_time(b) for a, b in ev]
    us = 1e3 * sorted(t)[len(t) // 2]
    feats = (p.n_q_heads + 2 * p.n_kv_heads) * p.head_dim
    flops = 2.0 * p.local_len * feats * hidden + 2.0 * p.local_len * hidden * p.n_kv_heads
    tf = flops / (us * 1e-6) / 1e12
    cpu = None
    if cpu_budget > 0:
        import oracle
        n_tok, el = 128, 0.0
        while True:  # local tokens scored by the oracle: doubled until the budget is spent
            rows = p.anchor_len + n_tok
            t0 = time.perf_counter()
            oracle.retaining_scores_ref(inp["q"][:, :rows], inp["k"][:, :rows], inp["v"][:, :rows],
                                        w["w1"], w["b1"], w["w2"], w["b2"], anchor_len=p.anchor_len)
            el = time.perf_counter() - t0
            if el > cpu_budget / 3 or n_tok * 2 > p.local_len:
                break
            n_tok *= 2
        f_s = 2.0 * n_tok * feats * hidden + 2.0 * n_tok * hidden * p.n_kv_heads
        cpu = {"value": round(f_s / el / 1e12, 6), "unit": "TFLOP/s", "cores": _oracle_threads(),
               "kind": "oracle", "sample": f"{n_tok} of {p.local_len} local tokens, fp64 NumPy; "
                                           f"{el:.1f} s wall"}
    return {"workload": wl.name, "local_len": p.local_len, "features": feats, "hidden": hidden,
            "n_kv_heads": p.n_kv_heads, "us": round(us, 2), "flops": flops,
            "tflops": round(tf, 1), "bound": "mfma", "peak": PEAK_BF16_TFLOPS,
            "frac": round(tf / PEAK_BF16_TFLOPS, 4),
            "kernel": "gemm_kernel<kXQkv, kWPlain, kEpiScorer> + scorer_reduce_kernel",
            "timing": f"median of {steps} back-to-back launches after at least 0.2 s of warm-up "
                      "launches, HIP events", "weights": "synthetic",
            "cpu_baseline": cpu}


def oracle_rows_rate(wl, inp, budget_s: float) -> dict:
    """fp64 oracle on a bounded sample of one workload: evenly spaced rows of
    query head 0 (doubled until the budget is spent), rated over those rows'
    visible (query, key) pairs; the whole share's oracle time is extrapolated
    from that rate and the share's unmasked FLOPs."""
    import numpy as np
    import oracle
    p = wl.problem
    n = 16
    while True:
        rows = np.unique(np.linspace(0, p.rows - 1, n).astype(np.int64))
        vis = np.where(rows < p.anchor_len, rows, rows + p.passing_rows) + 1
        flops = 4.0 * p.head_dim * float(vis.sum())
        t0 = time.perf_counter()
        oracle.attention_ref(inp["q"], inp["k"], inp["v"], inp["k_pass"], inp["v_pass"],
                             anchor_len=p.anchor_len, heads=np.array([0]), rows=rows)
        el = time.perf_counter() - t0
        if el > budget_s / 3 or n >= p.rows:
            break
        n *= 2
    rate = flops / el
    total = oracle.attention_flops(p.n_q_heads, p.head_dim, p.anchor_len, p.local_len,
                                   p.passing_rows)
    return {"value": round(rate / 1e12, 6), "unit": "TFLOP/s", "cores": _oracle_threads(),
            "kind": "oracle",
            "sample": f"{len(rows)} evenly spaced rows of query head 0 of {p.n_q_heads} heads x "
                      f"{p.rows} rows, fp64 NumPy, {el:.2f} s wall; the whole share's oracle time "
                      "is extrapolated from this rate",
            "oracle_s_extrapolated": round(total / rate, 1)}


def bench_workload_row(name: str, steps: int, warmup: int, seed: int = 0,
                       cpu_budget: float = 0.0) -> dict:
    """One host-share workload end to end (compressor, then attention, one
    stream), inputs resident in HBM, HIP events around each kernel on the
    launch stream; the attention time is the average launch."""
    import numpy as np
    import torch
    from paper_2502_12085_amd import apb, inputs

    wl = inputs.WORKLOADS[name]
    p = wl.problem
    print(f"# workload {name}: generating inputs", file=sys.stderr, flush=True)
    inp = inputs.make_inputs(wl, seed)

    def dev(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()

    q, k, v = dev(inp["q"]), dev(inp["k"]), dev(inp["v"])
    scores = torch.from_numpy(inp["scores"]).cuda()
    kbuf = torch.zeros((p.n_hosts, p.n_kv_heads, p.pass_len, p.head_dim), dtype=torch.bfloat16,
                       device="cuda")
    vbuf = torch.zeros_like(kbuf)
    if p.host_idx:
        kbuf[:p.host_idx] = dev(inp["k_pass"])
        vbuf[:p.host_idx] = dev(inp["v_pass"])
    idx = torch.empty((p.n_kv_heads, p.pass_len), dtype=torch.int32, device="cuda")
    o = torch.empty((p.n_q_heads, p.rows, p.head_dim), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((p.n_q_heads, p.rows), dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]

    def step(e=None):
        if e:
            e[0].record(stream)
        apb.compress_select(p, scores, k, v, idx, kbuf[p.host_idx], vbuf[p.host_idx], stream)
        if e:
            e[1].record(stream)
        apb.attention_fwd(p, q, k, v, kbuf, vbuf, o, lse, 0.0, stream)
        if e:
            e[2].record(stream)

    step_ms_warm = warm_up(step, warmup)
    if step_ms_warm < 1.0:
        busy_ahead(stream)  # few-microsecond steps: keep host gaps out of the events
    for e in ev:
        step(e)
    torch.cuda.synchronize()
    comp_us = 1e3 * sum(a.elapsed_time(b) for a, b, _ in ev) / steps
    attn_ms = sum(b.elapsed_time(c) for _, b, c in ev) / steps
    step_ms = sum(a.elapsed_time(c) for a, _, c in ev) / steps
    flops = apb.attention_flops(p)
    comp_bytes = (4 * p.n_kv_heads * p.local_len + 4 * p.n_kv_heads * p.pass_len
                  + 2 * 2 * p.n_kv_heads * p.pass_len * p.head_dim * 2)
    tf = flops / (attn_ms * 1e-3) / 1e12
    row = {"workload": name, "n_q_heads": p.n_q_heads, "n_kv_heads": p.n_kv_heads,
           "head_dim": p.head_dim, "anchor_len": p.anchor_len, "local_len": p.local_len,
           "pass_len": p.pass_len, "host_idx": p.host_idx, "n_hosts": p.n_hosts,
           "unmasked_flops": flops, "attention_ms": round(attn_ms, 4),
           "attention_tflops": round(tf, 1), "frac_of_peak": round(tf / PEAK_BF16_TFLOPS, 4),
           "compress_us": round(comp_us, 2),
           "compress_gbs": round(comp_bytes / (comp_us * 1e-6) / 1e9, 1),
           "step_ms": round(step_ms, 4),
           "tokens_per_s": round(p.rows / (step_ms * 1e-3), 1),
           "timing": f"average of {steps} back-to-back steps, HIP events per kernel"}
    if cpu_budget > 0:
        print(f"# workload {name}: oracle sample", file=sys.stderr, flush=True)
        row["cpu_baseline"] = oracle_rows_rate(wl, inp, cpu_budget)
    del q, k, v, o, lse, kbuf, vbuf, scores, idx, inp
    torch.cuda.empty_cache()
    return row


# The paper's headline speedups (whole-model serving speed, RULER/InfiniteBench
# style synthetic-length runs of Llama-3.1-8B, Table of speed against input
# length) and the hardware they were measured on; context only.
PAPER_SPEEDUPS = {
    "vs_flashattn": {"speedup": 9.2, "apb_tok_s": 37575, "other_tok_s": 4086, "context": "128K",
                     "hardware": "APB on 8x NVIDIA A800-80GB; FlashAttn on 1x A800-80GB"},
    "vs_ringattn": {"speedup": 4.2, "apb_tok_s": 26102, "other_tok_s": 6255, "context": "512K",
                    "hardware": "both on 8x NVIDIA A800-80GB"},
    "vs_starattn": {"speedup": 1.6, "apb_tok_s": 26102, "other_tok_s": 16177, "context": "512K",
                    "hardware": "both on 8x NVIDIA A800-80GB"},
    "note": "end-to-end tokens/s of the whole model over all hosts (input plus output tokens "
            "over prefill plus decode time); not comparable with this single-GPU host-share rate",
}


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="llama8b_128k")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--cpu-budget", type=float, default=20.0,
                    help="seconds of oracle work for cpu_baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-stage2", action="store_true",
                    help="skip the decoding-stage (Alg. 3) measurement")
    ap.add_argument("--no-scorer", action="store_true",
                    help="skip the retaining-head scorer measurement")
    ap.add_argument("--overlap", action="store_true",
                    help="run the compressor on a second stream, concurrent with the attention")
    ap.add_argument("--no-layer", action="store_true",
                    help="skip the whole-layer (Alg. 2) measurement")
    ap.add_argument("--no-ceiling", action="store_true",
                    help="skip the matrix-core ceiling probe")
    ap.add_argument("--no-workloads", action="store_true",
                    help="skip timing the other workloads (tiny, 32K, 256K, 512K)")
    ap.add_argument("--no-power", action="store_true",
                    help="skip reading socket power and shader clock under the attention kernel")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device-to-device copy of MIB MiB (for scaling "
                         "the HBM byte counters) and exit")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py runs one host share on one GPU; --gpus {args.gpus} is not supported "
              "(the multi-GPU all-gather of compressed blocks is not built).", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_2502_12085_amd import apb, inputs

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    if args.copy_calibration:
        n = args.copy_calibration << 20
        src = torch.ones(n // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(args.steps):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes_read": n, "bytes_written": n,
                          "launches": args.steps}), flush=True)
        return
    apb.lib()  # fail loudly now if the HIP library is missing

    wl = inputs.WORKLOADS[args.workload]
    p = wl.problem
    print(f"# generating {wl.name} inputs", file=sys.stderr, flush=True)
    inp = inputs.make_inputs(wl, args.seed)

    def dev(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()

    q, k, v = dev(inp["q"]), dev(inp["k"]), dev(inp["v"])
    scores = torch.from_numpy(inp["scores"]).cuda()
    # rank-major passing buffer [H][n_kv][l_p][d]: slots < host_idx hold the
    # earlier hosts' compressed blocks, slot host_idx receives this host's.
    kbuf = torch.zeros((p.n_hosts, p.n_kv_heads, p.pass_len, p.head_dim), dtype=torch.bfloat16,
                       device="cuda")
    vbuf = torch.zeros_like(kbuf)
    kbuf[:p.host_idx] = dev(inp["k_pass"])
    vbuf[:p.host_idx] = dev(inp["v_pass"])
    idx = torch.empty((p.n_kv_heads, p.pass_len), dtype=torch.int32, device="cuda")
    o = torch.empty((p.n_q_heads, p.rows, p.head_dim), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((p.n_q_heads, p.rows), dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()

    stream = torch.cuda.current_stream()
    # This host's compressor writes slot host_idx, which its own attention
    # does not read (it reads slots < host_idx): --overlap runs the
    # compressor on a second stream (default priority) concurrently with the
    # attention; by default they run back to back on one stream.
    side = torch.cuda.Stream()
    ev = [tuple(torch.cuda.Event(enable_timing=True) for _ in range(5))
          for _ in range(args.steps)]

    def step(events=None):
        start = events[0] if events else torch.cuda.Event()
        start.record(stream)
        cs = side if args.overlap else stream
        if args.overlap:
            cs.wait_event(start)
        if events:
            events[1].record(cs)
        apb.compress_select(p, scores, k, v, idx, kbuf[p.host_idx], vbuf[p.host_idx], cs)
        if events:
            events[2].record(cs)
            events[3].record(stream)
        apb.attention_fwd(p, q, k, v, kbuf, vbuf, o, lse, 0.0, stream)
        if events:
            events[4].record(stream)
        if args.overlap:
            stream.wait_stream(side)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(ev[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    # compressor with cold caches: a 1 GiB fill evicts L2 and the 256 MB
    # Infinity Cache before each timed launch
    flush = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
    cold = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
            for _ in range(args.steps)]
    for i, (c0, c1) in enumerate(cold):
        flush.fill_(float(i))
        c0.record(stream)
        apb.compress_select(p, scores, k, v, idx, kbuf[p.host_idx], vbuf[p.host_idx], stream)
        c1.record(stream)
    torch.cuda.synchronize()
    del flush
    cold_us = 1e3 * sorted(a.elapsed_time(b) for a, b in cold)[len(cold) // 2]

    comp_ms = [e[1].elapsed_time(e[2]) for e in ev]
    attn_ms = [e[3].elapsed_time(e[4]) for e in ev]
    ms_step = wall * 1e3 / args.steps
    flops = apb.attention_flops(p)
    attn_avg = sum(attn_ms) / len(attn_ms)
    achieved = flops / (attn_avg * 1e-3) / 1e12
    traffic = measured_traffic(wl.name)
    value = flops / (ms_step * 1e-3) / 1e12
    comp_bytes = (4 * p.n_kv_heads * p.local_len + 4 * p.n_kv_heads * p.pass_len
                  + 2 * 2 * p.n_kv_heads * p.pass_len * p.head_dim * 2)

    result = {
        "metric": "APB host-share prefill attention TFLOP/s",
        "value": round(value, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": wl.name, "n_hosts": p.n_hosts, "host_idx": p.host_idx,
                   "anchor_len": p.anchor_len, "local_len": p.local_len,
                   "pass_len": p.pass_len, "n_q_heads": p.n_q_heads,
                   "n_kv_heads": p.n_kv_heads, "head_dim": p.head_dim,
                   "outlier_k": wl.outlier_k, "zipf_scores": wl.zipf_scores},
        "pct_bf16_peak": round(100 * value / PEAK_BF16_TFLOPS, 2),
        "tokens_per_s": round(p.rows / (ms_step * 1e-3), 1),
        "attention_ms": round(attn_avg, 4),
        "step_schedule": ("compressor on a second stream, concurrent with the attention"
                          if args.overlap else "compressor then attention, one stream"),
        "compress_us": round(1e3 * sum(comp_ms) / len(comp_ms), 2),
        "compress_gbs": round(comp_bytes / (sum(comp_ms) / len(comp_ms) * 1e-3) / 1e9, 1),
        "compress_cold_us": round(cold_us, 2),
        "compress_cold_gbs": round(comp_bytes / (cold_us * 1e-6) / 1e9, 1),
        "unmasked_flops": flops,
        "roofline": {"bound": "mfma", "achieved": round(achieved, 3), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                     "traffic": traffic, "kernel": "attn_fwd_kernel<128>",
                     "kernel_source_hash": kernel_source_hash()},
        "paper_context": {"a800_attention_ms_per_block": 34.07,
                          "a800_implied_tflops": round(flops / 34.07e-3 / 1e12, 1),
                          "note": "8xA800 per-block breakdown at 128K; another machine",
                          "headline_speedups": PAPER_SPEEDUPS},
    }
    if not args.no_ceiling:
        ceil = bench_mfma_ceiling(max(args.steps // 2, 5))
        ceil["attention_frac_of_ceiling"] = round(achieved / ceil["tflops"], 4)
        result["mfma_ceiling"] = ceil
    if not args.no_layer and args.workload in ("llama8b_128k", "llama8b_32k"):
        print("# whole-layer measurement", file=sys.stderr, flush=True)
        result["layer"] = bench_layer(inputs.LAYER_WORKLOADS[args.workload + "_layer"],
                                      max(args.steps // 2, 5), 2)
    if not args.no_scorer:
        result["scorer"] = bench_scorer(wl, max(args.steps, 10), 3,
                                        cpu_budget=0.0 if args.no_cpu_baseline else 6.0)
    if not args.no_stage2:
        result["stage2"] = [bench_stage2(inputs.DECODE_WORKLOADS[n], max(args.steps, 20), 5,
                                         cpu_budget=0.0 if args.no_cpu_baseline else 3.0)
                            for n in ("llama8b_128k_decode", "llama8b_128k_question")]
    if not args.no_power:
        # last of the GPU legs on these inputs, so its seconds of full-power
        # load do not precede the timed ones
        result["power"] = sample_power(
            lambda: apb.attention_fwd(p, q, k, v, kbuf, vbuf, o, lse, 0.0, stream))
    if not args.no_cpu_baseline:
        print("# timing the fp64 oracle on the host cores", file=sys.stderr, flush=True)
        result["cpu_baseline"] = cpu_baseline(wl, inp, args.cpu_budget)
    if not args.no_workloads:
        # every workload in one record: this one from the measurement above,
        # the others timed here (fewer steps for the longest)
        rows = []
        del inp, q, k, v, o, lse, kbuf, vbuf, scores, idx
        torch.cuda.empty_cache()
        for name in inputs.WORKLOADS:
            if name == wl.name:
                rows.append({"workload": name, "unmasked_flops": flops,
                             "attention_ms": round(attn_avg, 4),
                             "attention_tflops": round(achieved, 1),
                             "frac_of_peak": round(achieved / PEAK_BF16_TFLOPS, 4),
                             "compress_us": result["compress_us"],
                             "compress_gbs": result["compress_gbs"],
                             "step_ms": round(ms_step, 4),
                             "tokens_per_s": result["tokens_per_s"],
                             "timing": "the headline measurement above",
                             "cpu_baseline": result.get("cpu_baseline")})
                continue
            big = inputs.WORKLOADS[name].problem.n_q_heads * inputs.WORKLOADS[name].problem.rows
            n_steps = 5 if big > 2_000_000 else max(args.steps // 2, 5)
            rows.append(bench_workload_row(name, n_steps, 2, args.seed,
                                           0.0 if args.no_cpu_baseline else 3.0))
        result["workloads"] = rows
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
