"""Throughput of the DBLast head + block draw + verification on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--settle-ms MS] [--workload qwen3_8b]
                    [--temperature T] [--mode soft|greedy|rows] [--no-cpu-baseline]
                    [--no-extras] [--copy-calibration BYTES]

One step is one pass of the whole hot path over one batch of synthetic inputs already resident
in HBM: dbl_head_logprobs (bf16 head GEMM + per-tile log-softmax), dbl_sample_block (category
and token draw) and dbl_verify_block (posterior, accept test, residual/bonus draw, acceptance
masses, AL_b and E). The Philox step counter advances every step. Before the W warm-up steps the
step runs untimed for --settle-ms of wall time (default 100), since the GPU's clock ramps for
~40 ms from idle; the line reports it under `settle`. Prints one JSON line; for the
Qwen3-8B workload it also carries the same step at the other target temperatures
(`temperature_sweep`) and the Qwen3-4B and stress workloads' steps (`other_workloads`), unless
--no-extras.
With --mode greedy the step is the greedy-branch variant: the head also returns each row's
argmax, then dbl_sample_greedy and dbl_verify_greedy.
With --mode rows the line instead times the other entry points at the workload's shape (branch
expander, prior head, objective forward, target transform, early-determinism estimate), each
against its own bound; it is a measurement aid, not the step metric.
With --workload objective (2048 blocks, R = 16) a step runs every 128-block chunk through the
head, dbl_expected_len and dbl_acceptance_objective.

The metric is verified block positions per second, B*K / step time. The roofline entry is for
the dominant kernel, the head GEMM: 2*M*d*V flops per launch over its average launch time,
measured with HIP events on the stream the library launches on, against MI355X's dense bf16
peak; `roofline.observed` adds the clock and MFMA busy fraction rocprofv3 measured on the same
head source (profiles/head_bf16_qwen3_8b_clock.json, written by --write-clock). The CPU baseline times the oracle (binary64 NumPy) on a bounded sample of the same
workload on this machine's host cores.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "verified block positions/sec at Qwen3-8B head shape; head-GEMM MFMA % of peak"
PEAK_BF16_TFLOPS = 2500.0        # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0            # MI355X HBM3E
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "head_bf16_qwen3_8b_traffic.json")
CLOCK_FILE = os.path.join(ROOT, "profiles", "head_bf16_qwen3_8b_clock.json")
N_SIMDS = 1024                   # MI355X: 256 CUs x 4 SIMDs
N_XCDS = 8
HEAD_SOURCE = os.path.join(ROOT, "paper_2608_05448_amd", "csrc", "head.hip")


def _head_source_hash() -> str:
    with open(HEAD_SOURCE, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def _traffic(workload: str):
    """HBM bytes per head launch from the committed rocprofv3 counter summary, or None when it
    is missing or was taken on a different head kernel source."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("head_source_sha256_16") != _head_source_hash() or rec.get("workload") != workload:
        return None
    return rec.get("hbm_bytes_per_launch")


def _clock(workload: str):
    """Observed clock and MFMA busy of the head kernel from the committed rocprofv3 record, or
    None when it is missing or was taken on a different head kernel source."""
    try:
        with open(CLOCK_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("head_source_sha256_16") != _head_source_hash() or rec.get("workload") != workload:
        return None
    return rec


def _write_clock(pmc_dir: str, workload: str):
    """Head clock and MFMA busy from one rocprofv3 run with --pmc GRBM_GUI_ACTIVE
    SQ_VALU_MFMA_BUSY_CYCLES and --kernel-trace: per head dispatch, GRBM_GUI_ACTIVE / 8 XCDs is
    the kernel's cycles, (end - start) its duration, and SQ_VALU_MFMA_BUSY_CYCLES / (1024 SIMDs x
    cycles) the MFMA pipes' busy fraction. The first dispatch (warm-up) is left out."""
    import csv
    import glob
    counters, spans = {}, {}
    for path in glob.glob(os.path.join(pmc_dir, "**", "*counter_collection.csv"), recursive=True):
        with open(path) as f:
            for row in csv.DictReader(f):
                if "head_bf16" in row["Kernel_Name"]:
                    d = counters.setdefault(row["Dispatch_Id"], {})
                    d[row["Counter_Name"]] = d.get(row["Counter_Name"], 0.0) + float(row["Counter_Value"])
    for path in glob.glob(os.path.join(pmc_dir, "**", "*kernel_trace.csv"), recursive=True):
        with open(path) as f:
            for row in csv.DictReader(f):
                if "head_bf16" in row["Kernel_Name"]:
                    spans[row["Dispatch_Id"]] = (int(row["End_Timestamp"]) - int(row["Start_Timestamp"]))
    ids = sorted((i for i in counters if i in spans), key=int)[1:]
    if not ids:
        raise SystemExit(f"no head dispatches with both counters and a trace under {pmc_dir}")
    cyc = sum(counters[i]["GRBM_GUI_ACTIVE"] / N_XCDS for i in ids) / len(ids)
    ns = sum(spans[i] for i in ids) / len(ids)
    busy = sum(counters[i]["SQ_VALU_MFMA_BUSY_CYCLES"] for i in ids) / len(ids)
    rec = {"workload": workload, "head_source_sha256_16": _head_source_hash(),
           "dispatches": len(ids), "head_us": ns / 1e3, "cycles": cyc,
           "clock_ghz": cyc / ns, "mfma_busy_cycles": busy,
           "mfma_busy": busy / (N_SIMDS * cyc)}
    with open(CLOCK_FILE, "w") as f:
        json.dump(rec, f, indent=1)
    print(json.dumps(rec))


def _cpu_baseline(wl, h, w, ell, logp, budget_s: float, mode: str = "soft"):
    """The oracle on as many whole blocks as fit the time budget (at least one)."""
    import numpy as np
    import torch
    from threadpoolctl import threadpool_info

    from oracle import greedy as GR
    from oracle import head as OH
    from oracle import mixture as MX

    ww = w.float().cpu().numpy()
    hh = h.float().cpu().numpy()
    ee = ell.cpu().numpy()
    lp = logp.cpu().numpy()
    K, R, d, V = wl.K, wl.R, wl.d, wl.V
    t0 = time.perf_counter()
    done = 0
    for b in range(wl.B):
        seq = np.array([b])
        if mode == "greedy":
            logits = OH.head_logits(hh[b].reshape(K * R, d), ww)
            xhat = GR.branch_tokens(logits).reshape(1, K, R)
            _, x = GR.sample_blocks_greedy(xhat, ee[b:b + 1], wl.z_temp, wl.philox_seed, 0, seq)
            GR.verify_blocks_greedy(xhat, ee[b:b + 1], wl.z_temp, x, lp[b:b + 1],
                                    wl.philox_seed, 0, seq)
        else:
            tls, lm, ls = OH.head_factored(hh[b].reshape(K * R, d), ww, v_chunk=8192)
            lq = OH.flat_logq(tls, lm, ls).reshape(1, K, R, V)
            _, x = MX.sample_blocks(tls.reshape(1, K, R, V), lm.reshape(1, K, R, -1),
                                    ls.reshape(1, K, R), ee[b:b + 1], wl.z_temp,
                                    wl.philox_seed, 0, seq)
            MX.verify_blocks(lq, ee[b:b + 1], wl.z_temp, x, lp[b:b + 1], wl.philox_seed, 0, seq)
        done += 1
        if time.perf_counter() - t0 >= budget_s:
            break
    el = time.perf_counter() - t0
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    cores = len(os.sched_getaffinity(0))
    return {"value": done * K / el, "unit": "positions/s", "cores": min(threads, cores),
            "kind": "oracle", "host": _host_cpu(),
            "sample": f"{done} of {wl.B} blocks ({done * K} positions): binary64 head, "
                      f"{'greedy-branch ' if mode == 'greedy' else ''}block draw and "
                      f"verification, {el:.1f} s on the host"}


def _host_cpu() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _cpu_baseline_objective(wl, h, w, ell, xs, logp, budget_s: float):
    """The oracle on whole blocks of one chunk of the objective workload (binary64 head, the
    expected length along the trajectory and the objective forward) until the time budget."""
    from threadpoolctl import threadpool_info

    from oracle import head as OH
    from oracle import mixture as MX
    from oracle import objective as OB

    ww = w.float().cpu().numpy()
    hh = h.float().cpu().numpy()
    ee = ell.cpu().numpy()
    xx = xs.cpu().numpy()
    lp = logp.cpu().numpy()
    K, R, d, V = wl.K, wl.R, wl.d, wl.V
    t0 = time.perf_counter()
    done = 0
    for b in range(len(xx)):
        tls, lm, ls = OH.head_factored(hh[b].reshape(K * R, d), ww, v_chunk=8192)
        lq = OH.flat_logq(tls, lm, ls).reshape(1, K, R, V)
        MX.expected_len_blocks(lq, ee[b:b + 1], wl.z_temp, xx[b:b + 1], lp[b:b + 1])
        OB.acceptance_objective(lq, ee[b:b + 1], wl.z_temp, xx[b:b + 1], lp[b:b + 1], tau=0.1)
        done += 1
        if time.perf_counter() - t0 >= budget_s:
            break
    el = time.perf_counter() - t0
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    return {"value": done * K / el, "unit": "positions/s",
            "cores": min(threads, len(os.sched_getaffinity(0))), "kind": "oracle",
            "host": _host_cpu(),
            "sample": f"{done} of {wl.B} blocks ({done * K} positions): binary64 head, expected "
                      f"length along the trajectory and objective forward, {el:.1f} s on the host"}


def _pmc_mean(csv_dir: str, counter: str, name_re: str) -> float:
    """Mean over dispatches (of kernels matching name_re) of a counter summed over instances."""
    import csv
    import glob
    import re
    per = {}
    for path in glob.glob(os.path.join(csv_dir, "*counter_collection.csv")):
        with open(path) as f:
            for row in csv.DictReader(f):
                if row["Counter_Name"] == counter and re.search(name_re, row["Kernel_Name"]):
                    per[row["Dispatch_Id"]] = per.get(row["Dispatch_Id"], 0.0) + float(
                        row["Counter_Value"])
    if not per:
        raise SystemExit(f"no {counter} rows for /{name_re}/ under {csv_dir}")
    return sum(per.values()) / len(per)


def _write_traffic(head_fetch, head_write, copy_fetch, copy_write, copy_bytes, workload):
    """HBM bytes per head launch from rocprofv3 FETCH_SIZE / WRITE_SIZE runs (KiB per dispatch),
    each scaled so that the same counter reads exactly copy_bytes for a plain device copy."""
    hf = _pmc_mean(head_fetch, "FETCH_SIZE", "head_bf16")
    hw = _pmc_mean(head_write, "WRITE_SIZE", "head_bf16")
    cf = _pmc_mean(copy_fetch, "FETCH_SIZE", "copyBuffer")
    cw = _pmc_mean(copy_write, "WRITE_SIZE", "copyBuffer")
    f_fetch = copy_bytes / (cf * 1024.0)
    f_write = copy_bytes / (cw * 1024.0)
    rec = {"workload": workload, "head_source_sha256_16": _head_source_hash(),
           "fetch_kib_per_launch": hf, "write_kib_per_launch": hw,
           "copy_bytes": copy_bytes, "copy_fetch_kib": cf, "copy_write_kib": cw,
           "fetch_scale": f_fetch, "write_scale": f_write,
           "hbm_read_bytes_per_launch": hf * 1024.0 * f_fetch,
           "hbm_write_bytes_per_launch": hw * 1024.0 * f_write,
           "hbm_bytes_per_launch": hf * 1024.0 * f_fetch + hw * 1024.0 * f_write}
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(rec, f, indent=1)
    print(json.dumps(rec))


def _copy_calibration(nbytes: int):
    """A plain device copy of known size, for scaling the FETCH_SIZE / WRITE_SIZE counters."""
    import torch
    n = nbytes // 4
    a = torch.ones(n, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": n * 4, "copy_bytes_written": n * 4, "launches": 3}))


def _rows(wl, dev, steps: int, warmup: int, cpu: bool = True):
    """Average time per call (HIP events on the library's stream) of the entry points outside
    the step, at the workload's shape, each with its algorithmic bytes or flops and bound; with
    ``cpu``, beside each the oracle's time on a bounded sample of the same call, scaled to the
    whole call."""
    import numpy as np
    import torch
    from threadpoolctl import threadpool_info

    import synth
    from paper_2608_05448_amd import dblast as D

    B, K, R, d, V = wl.B, wl.K, wl.R, wl.d, wl.V
    stream = torch.cuda.current_stream(dev)

    def timed(fn):
        for _ in range(warmup):
            fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize(dev)
        e0.record(stream)
        for _ in range(steps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize(dev)
        return e0.elapsed_time(e1) / steps

    def hbm(ms, nbytes):
        gbs = nbytes / (ms * 1e-3) / 1e9
        return {"ms": ms, "bound": "hbm", "bytes": nbytes, "achieved": gbs,
                "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": gbs / PEAK_HBM_GBS}

    def oracle(fn, scale, sample):
        t0 = time.perf_counter()
        fn()
        el = time.perf_counter() - t0
        threads = max([q.get("num_threads", 1) for q in threadpool_info()] + [1])
        return {"value": el * scale * 1e3, "unit": "ms per call (sample time x scale)",
                "cores": min(threads, len(os.sched_getaffinity(0))), "kind": "oracle",
                "sample": f"{sample}: {el * 1e3:.3f} ms on the host, x{scale:g}"}

    rows = {}
    # Branch expander: [B*K, d] x [R*d, d]^T plus bias and residual, bf16 out.
    ht = synth.make_uniform_logits((B, K, d), 11, device=dev).to(torch.bfloat16)
    We = (synth.make_uniform_logits((R * d, d), 12, device=dev) * (0.5 / d ** 0.5)).to(torch.bfloat16)
    ce = (synth.make_uniform_logits((R * d,), 13, device=dev) * 0.1).to(torch.bfloat16)
    hb = torch.empty((B, K, R, d), dtype=torch.bfloat16, device=dev)
    ms = timed(lambda: D.dbl_expand_branches(ht, We, ce, R, out=hb))
    r = hbm(ms, 2.0 * (R * d * d + B * K * d + R * d + B * K * R * d))
    r["tflops"] = 2.0 * B * K * R * d * d / (ms * 1e-3) / 1e12
    rows["expand_branches"] = r
    if cpu:
        from oracle import expander as EX
        h8 = ht.reshape(B * K, d)[:8].double().cpu().numpy()
        W64, c64 = We.double().cpu().numpy(), ce.double().cpu().numpy()
        r["cpu_baseline"] = oracle(lambda: EX.expand_branches(h8, W64, c64, round_bf16=True),
                                   B * K / 8, f"8 of {B * K} trunk rows")
    # Prior head: category logits from the anchor states.
    U = (synth.make_uniform_logits((R, d), 14, device=dev) * (1.0 / d ** 0.5)).to(torch.bfloat16)
    e = (synth.make_uniform_logits((R,), 15, device=dev) * 0.1).to(torch.bfloat16)
    pl = torch.empty((B, R), dtype=torch.float32, device=dev)
    ha = ht[:, 0].contiguous()
    ms = timed(lambda: D.dbl_prior_head(ha, U, e, out=pl))
    rows["prior_head"] = {"ms": ms, "bound": "latency"}
    if cpu:
        from oracle import expander as EX
        ha64, U64, e64 = ha.double().cpu().numpy(), U.double().cpu().numpy(), e.double().cpu().numpy()
        rows["prior_head"]["cpu_baseline"] = oracle(lambda: EX.prior_logits(ha64, U64, e64), 1,
                                                    f"all {B} blocks")
    # Objective forward along target trajectories (head outputs of the step's inputs).
    h = synth.make_h(wl, dev)
    w = synth.make_w(wl, dev)
    tls, lmass, lse = D.dbl_head_logprobs(h, w)
    del w
    ell = synth.make_ell(wl, dev)
    logp = synth.make_logp(wl, rows=K, device=dev)
    xs = synth.make_trajectory(wl, logp)
    ms = timed(lambda: D.dbl_acceptance_objective(tls, lmass, lse, ell, xs, logp, z_temp=wl.z_temp))
    rows["acceptance_objective"] = {"ms": ms, "bound": "latency", "blocks": B}
    del tls, lmass, lse
    if cpu:   # the oracle's own head output for one block (not timed), then its objective
        from oracle import head as OH
        from oracle import objective as OB
        w_np = synth.make_w(wl, dev).float().cpu().numpy()
        t_, l_, s_ = OH.head_factored(h[0].float().cpu().numpy().reshape(K * R, d), w_np,
                                      v_chunk=8192)
        del w_np
        lq1 = OH.flat_logq(t_, l_, s_).reshape(1, K, R, V)
        e1, x1, lp1 = ell[:1].cpu().numpy(), xs[:1].cpu().numpy(), logp[:1].cpu().numpy()
        rows["acceptance_objective"]["cpu_baseline"] = oracle(
            lambda: OB.acceptance_objective(lq1, e1, wl.z_temp, x1, lp1, tau=0.1), B,
            f"1 of {B} blocks (given the oracle head's log-probs)")
    del h
    # Target transform on the verification rows (K + 1 per block) with the paper's filters.
    g = synth.make_target_logits(wl, K + 1, device=dev).to(torch.float32)
    lp = torch.empty_like(g)
    nbytes = 2.0 * g.numel() * 4
    ws_t = torch.empty(D.dbl_workspace_bytes(D.DBL_OP_TARGET, B * (K + 1), 1, 1, 0, V),
                       dtype=torch.uint8, device=dev)
    for T, k, p in ((0.7, 20, 0.8), (1.0, 20, 0.95), (1.0, 0, 0.95)):
        ms = timed(lambda: D.dbl_target_logprobs(g, T, k, p, out=lp, ws=ws_t))
        rows[f"target_logprobs_T{T}_k{k}_p{p}"] = hbm(ms, nbytes)
        ms1 = timed(lambda: D.dbl_target_logprobs(g, T, k, p, out=lp, split=False))
        rows[f"target_logprobs_T{T}_k{k}_p{p}"]["ms_one_workgroup_per_row"] = ms1
        if cpu:
            from oracle import target as TG
            g4 = g.reshape(-1, V)[:4].cpu().numpy()
            rows[f"target_logprobs_T{T}_k{k}_p{p}"]["cpu_baseline"] = oracle(
                lambda: TG.filter_logprobs(g4, T, k, p), B * (K + 1) / 4,
                f"4 of {B * (K + 1)} rows")
    # Early determinism on the filtered rows.
    rng = np.random.default_rng(0)
    xd = torch.from_numpy(rng.integers(0, V, size=(B, K + 1), dtype=np.int32)).to(dev)
    ms = timed(lambda: D.dbl_early_determinism(xd, lp))
    rows["early_determinism"] = {"ms": ms, "bound": "latency", "blocks": B}
    if cpu:
        from oracle import target as TG
        lpx = np.log(np.random.default_rng(1).uniform(1e-3, 1.0, size=(B, K + 1)))
        rows["early_determinism"]["cpu_baseline"] = oracle(
            lambda: TG.early_determinism(lpx), 1, f"all {B} blocks (synthetic gathered log-probs)")
    # Reference rates for the streaming kernels, over as many bytes as the verify stream reads:
    # the library's plain streaming-read probe and a plain device copy.
    del g, lp
    buf = torch.empty(B * K * (R + 1) * V, dtype=torch.float32, device=dev).fill_(1.0)
    dst = torch.empty_like(buf)
    parts = torch.empty(2048, dtype=torch.float32, device=dev)
    ms = timed(lambda: D.dbl_stream_read_probe(buf, parts))
    rows["reference_read"] = hbm(ms, buf.numel() * 4.0)
    ms = timed(lambda: dst.copy_(buf))
    rows["reference_copy"] = hbm(ms, buf.numel() * 8.0)
    del buf, dst
    # Reference for the head: the vendor library's plain bf16 GEMM of the same shape (hipBLASLt
    # through torch's linear: logits = h w^T, bf16 output, no log-softmax), against the library
    # head (GEMM + fused per-tile log-softmax, fp32 output, LSE); at this workload's shape and,
    # for comparison, at the Qwen3-4B head's.
    def head_pair(hw, suffix):
        hB, hK, hR, hd, hV = hw.B, hw.K, hw.R, hw.d, hw.V
        hh = synth.make_h(hw, dev).reshape(hB * hK * hR, hd)
        ww = synth.make_w(hw, dev)
        logits = torch.empty((hB * hK * hR, hV), dtype=torch.bfloat16, device=dev)
        ms = timed(lambda: torch.matmul(hh, ww.t(), out=logits))
        flop = 2.0 * hB * hK * hR * hd * hV
        rows["reference_gemm" + suffix] = {
            "ms": ms, "bound": "mfma", "tflops": flop / (ms * 1e-3) / 1e12,
            "frac": flop / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
            "what": "torch.matmul (hipBLASLt), bf16 in and out, no epilogue"}
        del logits
        tls = torch.empty((hB, hK, hR, hV), dtype=torch.float32, device=dev)
        lmass = torch.empty((hB, hK, hR, D.ntiles(hV)), dtype=torch.float32, device=dev)
        lse = torch.empty((hB, hK, hR), dtype=torch.float32, device=dev)
        ms = timed(lambda: D.dbl_head_logprobs(hh.view(hB, hK, hR, hd), ww, tls, lmass, lse))
        rows["head_logprobs" + suffix] = {"ms": ms, "bound": "mfma",
                                          "tflops": flop / (ms * 1e-3) / 1e12,
                                          "frac": flop / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS}

    head_pair(wl, "")
    if wl.name != "qwen3_4b":
        head_pair(synth.WORKLOADS["qwen3_4b"], "_qwen3_4b")
    return {"metric": "per-call time of the entry points outside the step", "rows": rows,
            "steps": steps, "warmup": warmup, "data": "synthetic",
            "config": {"workload": wl.name, "B": B, "K": K, "R": R, "d": d, "V": V,
                       "target_rows": B * (K + 1)}}


def _objective_chunks(wl, dev, steps: int, warmup: int, chunk: int = 128, cpu: bool = True,
                      cpu_budget: float = 12.0):
    """The training-objective workload (2048 blocks, R = 16): one step runs every chunk of
    `chunk` blocks through dbl_head_logprobs, dbl_expected_len (β and E along the target
    trajectory) and dbl_acceptance_objective, with all chunks' inputs resident in HBM."""
    import torch

    import synth
    from paper_2608_05448_amd import dblast as D

    B, K, R, d, V = wl.B, wl.K, wl.R, wl.d, wl.V
    nT = D.ntiles(V)
    w = synth.make_w(wl, dev)
    ell = synth.make_ell(wl, dev)
    chunks = []
    for c0 in range(0, B, chunk):
        blocks = range(c0, min(B, c0 + chunk))
        lp = synth.make_logp(wl, rows=K, device=dev, blocks=blocks)
        chunks.append((synth.make_h(wl, dev, blocks=blocks), lp, synth.make_trajectory(wl, lp, blocks),
                       ell[c0:c0 + len(blocks)].contiguous()))
    nb = len(chunks[0][2])
    tls = torch.empty((nb, K, R, V), dtype=torch.float32, device=dev)
    lmass = torch.empty((nb, K, R, nT), dtype=torch.float32, device=dev)
    lse = torch.empty((nb, K, R), dtype=torch.float32, device=dev)
    beta = torch.empty((nb, K), dtype=torch.float32, device=dev)
    e = torch.empty(nb, dtype=torch.float32, device=dev)
    ws = torch.empty(D.dbl_workspace_bytes(D.DBL_OP_EXPECTED_LEN, nb, K, R, d, V),
                     dtype=torch.uint8, device=dev)
    obj = {k: torch.empty(nb, dtype=t, device=dev)
           for k, t in (("ell_tau", torch.int32), ("J", torch.float32), ("nll", torch.float32))}
    stream = torch.cuda.current_stream(dev)
    ev = []

    def step(record):
        for h, lp, xs, el in chunks:
            if len(xs) != nb:
                raise ValueError("the block count must be a multiple of the chunk size")
            e0, e1, e2, e3 = (torch.cuda.Event(enable_timing=True) for _ in range(4))
            if record:
                e0.record(stream)
            D.dbl_head_logprobs(h, w, tls, lmass, lse)
            if record:
                e1.record(stream)
            D.dbl_expected_len(tls, lmass, lse, el, xs, lp, z_temp=wl.z_temp, beta=beta,
                               exp_len=e, ws=ws)
            if record:
                e2.record(stream)
            D.dbl_acceptance_objective(tls, lmass, lse, el, xs, lp, z_temp=wl.z_temp, tau=0.1,
                                       want_terms=False, out=obj)
            if record:
                e3.record(stream)
                ev.append((e0, e1, e2, e3))

    for _ in range(warmup):
        step(False)
    torch.cuda.synchronize(dev)
    t0 = time.perf_counter()
    for _ in range(steps):
        step(True)
    torch.cuda.synchronize(dev)
    wall = time.perf_counter() - t0
    n = len(ev)
    head_ms = sum(a.elapsed_time(b) for a, b, _, _ in ev) / n
    el_ms = sum(b.elapsed_time(c) for _, b, c, _ in ev) / n
    ob_ms = sum(c.elapsed_time(d_) for _, _, c, d_ in ev) / n
    step_ms = ev[0][0].elapsed_time(ev[-1][3]) / steps
    M = nb * K * R
    head_tflops = 2.0 * M * d * V / (head_ms * 1e-3) / 1e12
    el_bytes = nb * K * (R + 1) * V * 4.0
    # Reference after the timed steps: the vendor library's plain bf16 GEMM at the chunk's head
    # shape (torch.matmul, hipBLASLt, bf16 output, no log-softmax), one chunk's h against w.
    h0 = chunks[0][0].reshape(M, d)
    logits = torch.empty((M, V), dtype=torch.bfloat16, device=dev)
    torch.matmul(h0, w.t(), out=logits)
    r0, r1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    r0.record(stream)
    for _ in range(3):
        torch.matmul(h0, w.t(), out=logits)
    r1.record(stream)
    torch.cuda.synchronize(dev)
    ref_ms = r0.elapsed_time(r1) / 3
    del logits
    ref_tflops = 2.0 * M * d * V / (ref_ms * 1e-3) / 1e12
    return {"metric": "positions/s of head + expected length + objective forward",
            "value": B * K / (step_ms * 1e-3), "unit": "positions/s", "n_gpus": 1,
            "steps": steps, "warmup": warmup, "ms_per_step": step_ms, "higher_is_better": True,
            "dtype": "bf16", "data": "synthetic",
            "config": {"workload": wl.name, "B": B, "K": K, "R": R, "d": d, "V": V,
                       "chunk_blocks": nb, "chunks": len(chunks)},
            "per_chunk_ms": {"head": head_ms, "expected_len": el_ms, "objective": ob_ms},
            "roofline": {"bound": "mfma", "achieved": head_tflops, "peak": PEAK_BF16_TFLOPS,
                         "unit": "TFLOP/s", "frac": head_tflops / PEAK_BF16_TFLOPS,
                         "kernel": "dbl_head_logprobs"},
            "reference_gemm_chunk": {"ms": ref_ms, "tflops": ref_tflops,
                                     "frac": ref_tflops / PEAK_BF16_TFLOPS,
                                     "what": "torch.matmul (hipBLASLt), bf16 in and out, no "
                                             "epilogue, one chunk's head shape"},
            "hbm": {"expected_len_GBps": el_bytes / (el_ms * 1e-3) / 1e9,
                    "expected_len_frac": el_bytes / (el_ms * 1e-3) / 1e9 / PEAK_HBM_GBS},
            "quality": {"mean_exp_len_last_chunk": float(e.mean().item()),
                        "mean_J_last_chunk": float(obj["J"].mean().item())},
            "wall_s_timed": wall,
            **({"cpu_baseline": _cpu_baseline_objective(wl, chunks[0][0], w, chunks[0][3],
                                                        chunks[0][2], chunks[0][1], cpu_budget)}
               if cpu else {})}


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--settle-ms", type=float, default=100.0,
                    help="untimed steps for at least this much wall time before the warm-up "
                         "steps, so the clock is at its sustained level (0: none)")
    ap.add_argument("--workload", default="qwen3_8b")
    ap.add_argument("--temperature", type=float, default=None)
    ap.add_argument("--mode", choices=("soft", "greedy", "rows"), default="soft")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the temperature sweep and the other step workloads")
    ap.add_argument("--cpu-budget", type=float, default=12.0)
    ap.add_argument("--copy-calibration", type=int, default=0)
    ap.add_argument("--write-clock", metavar="PMC_DIR",
                    help="turn a rocprofv3 --pmc GRBM_GUI_ACTIVE SQ_VALU_MFMA_BUSY_CYCLES "
                         "--kernel-trace run into the committed head clock record (no GPU work)")
    ap.add_argument("--write-traffic", nargs=5, metavar=("HEAD_FETCH_DIR", "HEAD_WRITE_DIR",
                                                         "COPY_FETCH_DIR", "COPY_WRITE_DIR",
                                                         "COPY_BYTES"),
                    help="turn rocprofv3 FETCH_SIZE/WRITE_SIZE CSV output into the committed "
                         "per-launch traffic record (no GPU work)")
    args = ap.parse_args(argv)

    if args.write_clock:
        _write_clock(args.write_clock, args.workload)
        return 0
    if args.write_traffic:
        hf, hw, cf, cw, nb = args.write_traffic
        _write_traffic(hf, hw, cf, cw, int(nb), args.workload)
        return 0

    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported (the hot "
              "path shards over blocks with no exchange; see the multi-GPU design notes)",
              file=sys.stderr)
        return 2

    import torch

    import synth
    from paper_2608_05448_amd import dblast as D

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    if args.copy_calibration:
        _copy_calibration(args.copy_calibration)
        return 0

    wl = synth.WORKLOADS[args.workload]
    if args.temperature is not None:
        wl = wl.replace(temperature=args.temperature)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    D.load()
    if args.mode == "rows":
        print(json.dumps(_rows(wl, dev, args.steps, args.warmup, not args.no_cpu_baseline)),
              flush=True)
        return 0
    if wl.name == "objective":
        print(json.dumps(_objective_chunks(wl, dev, args.steps, args.warmup,
                                           cpu=not args.no_cpu_baseline,
                                           cpu_budget=args.cpu_budget)), flush=True)
        return 0

    head = _step_run(wl, dev, args.mode, args.steps, args.warmup, settle_ms=args.settle_ms)
    B, K, R, d, V = wl.B, wl.K, wl.R, wl.d, wl.V
    step_ms = head["ms_per_step"]
    M = B * K * R
    head_ms = head["kernels_ms"]["head"]
    head_tflops = 2.0 * M * d * V / (head_ms * 1e-3) / 1e12
    traffic = _traffic(args.workload) if args.mode == "soft" else None
    roofline = {"bound": "mfma", "achieved": head_tflops, "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": head_tflops / PEAK_BF16_TFLOPS, "traffic": traffic,
                "kernel": "dbl_head_logprobs (head GEMM + per-tile log-softmax, LSE)",
                "flop_per_launch": 2.0 * M * d * V}
    clock = _clock(args.workload) if args.mode == "soft" else None  # taken on the soft head
    if clock is not None:
        # The 2.5 PFLOP/s peak assumes 2.4 GHz; under this load the clock is lower. All of these
        # come from the profiled run (counters on), whose head time is its own; the clock this
        # run's head implies follows from the same cycle count over this run's time.
        peak_at_clock = PEAK_BF16_TFLOPS * clock["clock_ghz"] / 2.4
        prof_tflops = 2.0 * M * d * V / (clock["head_us"] * 1e-6) / 1e12
        roofline["observed"] = {"clock_ghz": clock["clock_ghz"],
                                "mfma_busy": clock["mfma_busy"],
                                "head_ms_profiled": clock["head_us"] / 1e3,
                                "peak_at_clock_tflops": peak_at_clock,
                                "frac_of_peak_at_clock": prof_tflops / peak_at_clock,
                                "clock_ghz_implied_here": clock["cycles"] / (head_ms * 1e6),
                                "source": os.path.relpath(CLOCK_FILE, ROOT)}
    out = {
        "metric": METRIC,
        "value": head["value"],
        "unit": "positions/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": step_ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": args.workload, "B": B, "K": K, "R": R, "d": d, "V": V,
                   "global_batch": B, "positions_per_step": B * K,
                   "target_temperature": wl.temperature, "z_temp": wl.z_temp,
                   "mode": args.mode, "parallelism": "single GPU"},
        "roofline": roofline,
        "kernels_ms": head["kernels_ms"],
        "step_ms_p10_p50_p90": head["step_ms_p10_p50_p90"],
        "hbm": head["hbm"],
        "quality": head["quality"],
        "wall_s_timed": head["wall_s_timed"],
        "settle": head["settle"],
    }
    if not args.no_extras and args.mode == "soft" and args.workload == "qwen3_8b":
        # The same step at the other target temperatures of the workload, and the step of the
        # Qwen3-4B and stress workloads (each with fewer timed steps); the headline is above.
        n = max(5, args.steps // 2)
        out["temperature_sweep"] = {}
        for T in synth.QWEN3_8B_TEMPERATURES:
            if T == wl.temperature:
                continue
            r = _step_run(wl.replace(temperature=T), dev, "soft", n, 3, with_inputs=True)
            out["temperature_sweep"][str(T)] = {k: r[k] for k in ("value", "ms_per_step",
                                                                  "kernels_ms", "quality")}
        out["other_workloads"] = {}
        for name in ("qwen3_4b", "stress"):
            ow = synth.WORKLOADS[name]
            r = _step_run(ow, dev, "soft", n, 3)
            r.pop("wall_s_timed", None)
            r.pop("settle", None)
            ohead = r["kernels_ms"]["head"]
            r["config"] = {"B": ow.B, "K": ow.K, "R": ow.R, "d": ow.d, "V": ow.V,
                           "target_temperature": ow.temperature}
            r["head_frac_of_bf16_peak"] = (2.0 * ow.B * ow.K * ow.R * ow.d * ow.V /
                                           (ohead * 1e-3) / 1e12 / PEAK_BF16_TFLOPS)
            out["other_workloads"][name] = r
    if not args.no_cpu_baseline:
        h, w, ell, logp = _inputs(wl, dev)
        out["cpu_baseline"] = _cpu_baseline(wl, h, w, ell, logp, args.cpu_budget, args.mode)
    print(json.dumps(out), flush=True)
    return 0


_INPUT_CACHE = {}


def _inputs(wl, dev):
    """Synthetic inputs of a workload, resident in HBM (kept for the process: the temperature
    sweep reuses the branch states and weights and regenerates only the target)."""
    import synth
    key = (wl.name, wl.temperature)
    if key not in _INPUT_CACHE:
        base = next((v for k, v in _INPUT_CACHE.items() if k[0] == wl.name), None)
        if base is None:
            if any(k[0] != wl.name for k in _INPUT_CACHE):
                _INPUT_CACHE.clear()
            h, w, ell = synth.make_h(wl, dev), synth.make_w(wl, dev), synth.make_ell(wl, dev)
        else:
            h, w, ell = base[:3]
        _INPUT_CACHE[key] = (h, w, ell, synth.make_logp(wl, rows=wl.K + 1, device=dev))
    return _INPUT_CACHE[key]


def _step_run(wl, dev, mode, steps, warmup, with_inputs=False, settle_ms=0.0):
    """Time `steps` steps (after `warmup`) of head + draw + verification on the workload, with
    HIP events on the library's stream; inputs resident in HBM before timing."""
    import torch

    from paper_2608_05448_amd import dblast as D

    h, w, ell, logp = _inputs(wl, dev)
    B, K, R, d, V = wl.B, wl.K, wl.R, wl.d, wl.V
    nT = D.ntiles(V)
    tls = torch.empty((B, K, R, V), dtype=torch.float32, device=dev)
    lmass = torch.empty((B, K, R, nT), dtype=torch.float32, device=dev)
    lse = torch.empty((B, K, R), dtype=torch.float32, device=dev)
    z = torch.empty(B, dtype=torch.int32, device=dev)
    x = torch.empty((B, K), dtype=torch.int32, device=dev)
    vout = {"n_accept": torch.empty(B, dtype=torch.int32, device=dev),
            "next_token": torch.empty(B, dtype=torch.int32, device=dev),
            "accept_mass": torch.empty((B, K), dtype=torch.float32, device=dev),
            "al_expected": torch.empty(B, dtype=torch.float32, device=dev),
            "exp_len": torch.empty(B, dtype=torch.float32, device=dev)}
    ws_s = torch.empty(D.dbl_workspace_bytes(D.DBL_OP_SAMPLE, B, K, R, d, V), dtype=torch.uint8,
                       device=dev)
    ws_v = torch.empty(D.dbl_workspace_bytes(D.DBL_OP_VERIFY, B, K, R, d, V), dtype=torch.uint8,
                       device=dev)
    greedy = mode == "greedy"
    am = torch.empty((B, K, R), dtype=torch.int32, device=dev)
    ws_h = torch.empty(D.dbl_workspace_bytes(D.DBL_OP_HEAD, B, K, R, d, V), dtype=torch.uint8,
                       device=dev)
    ws_g = torch.empty(D.dbl_workspace_bytes(D.DBL_OP_VERIFY_GREEDY, B, K, R, d, V),
                       dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream(dev)

    def step(t, ev=None):
        if ev is not None:
            ev[0].record(stream)
        if greedy:
            D.dbl_head_logprobs(h, w, tls, lmass, lse, argmax=am, ws=ws_h)
        else:
            D.dbl_head_logprobs(h, w, tls, lmass, lse)
        if ev is not None:
            ev[1].record(stream)
        if greedy:
            D.dbl_sample_greedy(am, ell, z_temp=wl.z_temp, seed=wl.philox_seed, step=t, V=V,
                                z_out=z, x_out=x)
        else:
            D.dbl_sample_block(tls, lmass, lse, ell, z_temp=wl.z_temp, seed=wl.philox_seed,
                               step=t, z_out=z, x_out=x, ws=ws_s)
        if ev is not None:
            ev[2].record(stream)
        if greedy:
            D.dbl_verify_greedy(am, ell, x, logp, z_temp=wl.z_temp, seed=wl.philox_seed, step=t,
                                out=vout, ws=ws_g)
        else:
            D.dbl_verify_block(tls, lmass, lse, ell, x, logp, z_temp=wl.z_temp,
                               seed=wl.philox_seed, step=t, out=vout, ws=ws_v)
        if ev is not None:
            ev[3].record(stream)

    # From idle the GPU's clock takes ~40 ms of this load to reach its sustained level (per-step
    # time 3.7 ms at the first step, 2.55 ms at the sixth, steady from about the seventeenth at
    # the Qwen3-8B shape), so before the warm-up steps the step runs for at least settle_ms of
    # wall time; the line reports how many steps that took.
    settle_steps = 0
    t_settle = time.perf_counter()
    while (time.perf_counter() - t_settle) * 1e3 < settle_ms:
        for _ in range(4):
            step(settle_steps)
            settle_steps += 1
        torch.cuda.synchronize(dev)
    for t in range(warmup):
        step(t)
    torch.cuda.synchronize(dev)
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]
    torch.cuda.synchronize(dev)
    t_wall = time.perf_counter()
    for i in range(steps):
        step(warmup + i, events[i])
    torch.cuda.synchronize(dev)
    wall = time.perf_counter() - t_wall

    head_ms = sum(e[0].elapsed_time(e[1]) for e in events) / steps
    sample_ms = sum(e[1].elapsed_time(e[2]) for e in events) / steps
    verify_ms = sum(e[2].elapsed_time(e[3]) for e in events) / steps
    step_ms = events[0][0].elapsed_time(events[-1][3]) / steps
    per_step = sorted(e[0].elapsed_time(e[3]) for e in events)
    pct = {q: per_step[min(len(per_step) - 1, int(q / 100 * len(per_step)))] for q in (10, 50, 90)}
    # Algorithmic bytes: soft verify streams R branch rows + the target row per position; the
    # soft draw reads, per position, the drawn branch row's tile masses and one 128-id tile
    # (latency-bound). Greedy verify streams one target row per block (the first rejected
    # position or the bonus row); the greedy draw reads no vocabulary row.
    verify_bytes = B * V * 4.0 if greedy else B * K * (R + 1) * V * 4.0
    sample_bytes = 0.0 if greedy else B * K * (D.ntiles(V) + 128) * 4.0
    return {
        "value": B * K / (step_ms * 1e-3),
        "ms_per_step": step_ms,
        "kernels_ms": {"head": head_ms, "sample": sample_ms, "verify": verify_ms},
        "step_ms_p10_p50_p90": [pct[10], pct[50], pct[90]],
        "hbm": {"verify_GBps": verify_bytes / (verify_ms * 1e-3) / 1e9,
                "verify_frac": verify_bytes / (verify_ms * 1e-3) / 1e9 / PEAK_HBM_GBS,
                "verify_bytes": verify_bytes,
                "sample_bytes": sample_bytes,
                "sample_bound": "latency"},
        "quality": {"mean_n_accept": float(vout["n_accept"].float().mean().item()),
                    "mean_exp_len": float(vout["exp_len"].float().mean().item()),
                    "mean_al_expected": float(vout["al_expected"].float().mean().item())},
        "wall_s_timed": wall,
        "settle": {"ms": settle_ms, "steps": settle_steps},
    }


if __name__ == "__main__":
    sys.exit(main())
