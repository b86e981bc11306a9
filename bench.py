"""Throughput of the sparsity-aware fused attention forward on one MI355X.

    python bench.py [--steps 50] [--warmup 25] [--workload NAME | --all]

One step is one whole ``steel_attn_fwd`` call -- live-block index build plus
the fused attention pass -- over one batch of synthetic inputs already
resident in HBM.  Protocol as in the paper's evaluation (Section V-A): 25
warm-up calls, then the mean over 50 timed calls; before them the same call
keeps the GPU busy for 0.5 s (``--clock-warmup``), because the chip raises
its clock over the first tenths of a second of load.

Metric: effective TFLOP/s counted on live 64x64 tiles only,
4 * 64 * 64 * D * N_live / t (QK^T and PV, a multiply-add counted as 2; the
softmax is not counted), and the dense-equivalent 4 * B * Hq * S_q * S_k * D / t,
both against the MI355X bf16 dense MFMA peak of 256 CU x 2.4 GHz x 4096
flop/clk/CU = 2516.6 TFLOP/s (AMD's published 2.5 PFLOP/s).

The roofline object is for the attention kernels alone: the same pass split
into plan (index) + run (attention), with HIP events around the run on the
stream it is launched on.  ``traffic`` is the HBM bytes per run measured with
rocprofv3 counters (recorded in profiles/attn_traffic.json together with the
hash of the kernel source they were taken on; null when the source changed).

The CPU baseline times the float64 oracle on the host cores on a bounded
sample of the same workload (whole query blocks of several heads, for about
--cpu-seconds seconds) and reports it in the same unit.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

METRIC = "effective attention TFLOP/s (live blocks) + % bf16 MFMA peak, 1×MI355X"
DEFAULT_WORKLOAD = "gqa32x8_s16384_d128_window1024_sink64"
PEAK_TFLOPS = 256 * 2.4e9 * 4096 / 1e12     # 2516.6
HBM_PEAK_GBS = 8000.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "attn_traffic.json")
KERNEL_SRCS = [os.path.join(ROOT, "paper_2607_09385_amd", "csrc", f)
               for f in ("attn_common.h", "attn_fwd.hip", "attn_ws.hip", "block_index.hip")]


def live_tile_counts(mask, B, Hq, S_q, S_k, causal, blk=64):
    """Live tiles per (b, h, qb): mask byte set and not entirely above the
    causal diagonal.  Used only to count the flops of the metric."""
    nQB, nKB = -(-S_q // blk), -(-S_k // blk)
    qb = np.arange(nQB)[:, None]
    kb = np.arange(nKB)[None, :]
    last_row = np.minimum((qb + 1) * blk, S_q) - 1
    alive = np.ones((nQB, nKB), dtype=bool)
    if causal:
        alive &= ~(kb * blk > last_row + (S_k - S_q))
    bits = np.ones((B, Hq, nQB, nKB), dtype=bool) if mask is None else (np.asarray(mask) != 0)
    return (bits & alive[None, None]).sum(-1)          # [B, Hq, nQB]


def kernel_hash():
    """Hash of the attention kernels' sources and of the index build (whose
    work order sets which tiles each XCD's L2 sees together): counter readings
    taken on other sources are not reported."""
    h = hashlib.sha256()
    for path in KERNEL_SRCS:
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def traffic_for(workload):
    """HBM bytes per attention run from committed rocprofv3 counter readings,
    or None when they are missing or were taken on another kernel source."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    entry = rec.get("workloads", {}).get(workload)
    if not entry or rec.get("kernel_sha") != kernel_hash():
        return None
    return entry.get("bytes_per_run")


# Softmax work per element of a live tile: one exp2, the fma that forms its
# argument, and half each of a 3-input max, a packed bf16 conversion and a bf16
# dot2 for the row sum.  Cycles per 64-lane instruction measured by
# `bench.py --mfma-peak` (steel_valu_rate, shader clock, from the first wave's
# start to the last wave's end): a SIMD with eight resident waves sustains
# v_exp_f32 every 5.26 cycles and v_fma_f32 every 1.98, while a single wave
# issues them only every 12.0 and 8.5 cycles (the other three instructions are
# taken at the fma's rate).
VALU_CYCLES_SIMD = 5.26 + 1.98 + 1.5 * 1.98       # per 64 elements, SIMD throughput
VALU_CYCLES_ONE_WAVE = 12.0 + 8.5 + 1.5 * 8.5     # per 64 elements, issued by one wave


def valu_bound(n_live, D):
    """The softmax alone on all 1,024 SIMDs at 2.4 GHz: at the SIMD's VALU
    throughput (the plain-ALU bound beside the MFMA one), and issued by one
    wave per SIMD at the single-wave rate together with that wave's own score
    MFMAs, which hold its issue (the structure of the wave-specialised kernel,
    whose one S-wave per head computes the scores and the softmax of 64 rows)."""
    elems = n_live * 64 * 64
    us = elems * VALU_CYCLES_SIMD / 64 / (256 * 4 * 2.4e9) * 1e6
    one = (elems * VALU_CYCLES_ONE_WAVE / 64 + n_live * (D // 4) * 32) / (256 * 4 * 2.4e9) * 1e6
    return {"bound": "alu", "us": round(us, 1),
            "model": "per live element: exp2 + fma + half max3 + half cvt_pk_bf16 + half dot2 at the measured "
                     "SIMD rates (v_exp_f32 5.26, v_fma_f32 1.98 cycles per 64 lanes)",
            "one_wave_softmax_us": round(one, 1),
            "one_wave_model": "same instructions issued by one wave per SIMD (v_exp_f32 every 12.0, others every "
                              "8.5 cycles) plus that wave's D/4 score MFMAs per tile (32 cycles each)",
            "mfma_us_at_peak": round(4.0 * 64 * 64 * D * n_live / PEAK_TFLOPS / 1e6, 1)}


def blas_threads():
    try:
        from threadpoolctl import threadpool_info
        n = [i.get("num_threads", 0) for i in threadpool_info() if i.get("user_api") == "blas"]
        if n:
            return max(n)
    except Exception:
        pass
    return len(os.sched_getaffinity(0))


def cpu_model():
    """The host CPU's model name, from /proc/cpuinfo."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(cfg, q, k, v, mask, counts, seconds):
    """Time the float64 oracle on groups of 16 whole query blocks, cycling over
    heads, until ``seconds`` have passed; report live TFLOP/s of what it
    covered (the oracle itself computes full score rows)."""
    import oracle
    rng = np.random.default_rng(1)
    groups = [(h, g0) for g0 in range(0, cfg.nQB, 16) for h in range(cfg.Hq)]
    order = rng.permutation(len(groups))
    done_rows, live_flops, n_groups = 0, 0.0, 0
    t0 = time.perf_counter()
    for gi in order:
        h, g0 = groups[gi]
        qbs = np.arange(g0, min(g0 + 16, cfg.nQB))
        rows = np.arange(g0 * 64, min((g0 + 16) * 64, cfg.S_q))
        idx = np.stack([np.zeros_like(rows), np.full_like(rows, h), rows], 1)
        oracle.attention_rows(q, k, v, idx, mask, cfg.scale, cfg.causal, 64)
        done_rows += rows.size
        per_qb_rows = np.bincount(rows // 64 - g0, minlength=qbs.size)
        live_flops += float((counts[0, h, qbs] * per_qb_rows).sum()) * 4 * 64 * cfg.D
        n_groups += 1
        if time.perf_counter() - t0 >= seconds:
            break
    el = time.perf_counter() - t0
    return {
        "value": live_flops / el / 1e12,
        "unit": "TFLOP/s",
        "cores": blas_threads(),
        "cpu_model": cpu_model(),
        "kind": "oracle",
        "sample": (f"{done_rows} query rows ({n_groups} groups of 16 query blocks of one head, "
                   f"random order) of the same workload, float64, full score rows; {el:.1f} s"),
        "seconds": el,
    }


def mfma_peak(iters=400000, waves_per_wg=4):
    """Achievable rate of v_mfma_f32_32x32x16_bf16 (the instruction of both
    attention products) on this chip, for constant and for N(0,1) operands:
    the chip lowers its clock under the matrix cores' data-dependent power
    draw, so this is the context for the roofline fraction, whose
    denominator stays the published peak.  One workgroup of waves_per_wg
    waves per CU; the average clock comes from the kernel's own counters
    (shader cycles over 100 MHz reference ticks)."""
    import torch
    from paper_2607_09385_amd import _lib
    lib = _lib.load()
    dev = torch.device("cuda:0")
    grid = 256
    sink = torch.empty(grid * 64 * waves_per_wg, dtype=torch.float32, device=dev)
    clocks = torch.zeros(2 * grid, dtype=torch.int64, device=dev)
    stream = torch.cuda.current_stream()
    g = torch.Generator().manual_seed(0)
    res = {"instruction": "v_mfma_f32_32x32x16_bf16", "grid": grid, "waves_per_cu": waves_per_wg,
           "iters": iters}
    for kind in ("constant", "normal"):
        if kind == "constant":
            ops = torch.ones((8, 64, 8), dtype=torch.bfloat16)
        else:
            ops = torch.randn((8, 64, 8), generator=g).to(torch.bfloat16)
        ops = ops.to(dev)

        def launch(n):
            st = lib.steel_mfma_peak(ops.data_ptr(), n, grid, waves_per_wg, sink.data_ptr(),
                                     clocks.data_ptr(), stream.cuda_stream)
            if st != 0:
                raise RuntimeError(f"steel_mfma_peak failed ({st})")
        launch(iters // 4)   # clock ramp
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        launch(iters)
        e1.record(stream)
        torch.cuda.synchronize()
        t = e0.elapsed_time(e1) / 1e3
        flops = grid * waves_per_wg * iters * 16 * 2.0 * 32 * 32 * 16
        c = clocks.view(grid, 2).cpu().double()
        ghz = float((c[:, 0] / (c[:, 1] / 100e6)).mean() / 1e9)
        res[kind] = {"tflops": round(flops / t / 1e12, 1), "frac_of_peak": round(flops / t / 1e12 / PEAK_TFLOPS, 3),
                     "ms": round(t * 1e3, 2), "avg_clock_ghz": round(ghz, 3)}
    res["valu"] = {name: [valu_rate(op, waves_per_wg=w, grid=g)
                          for w, g in ((4, 256), (8, 256), (16, 256), (16, 512))]
                   for op, name in ((0, "v_exp_f32"), (1, "v_fma_f32"))}
    res["lds"] = {name: [lds_rate(op, waves_per_cu=w) for w in (4, 8, 16)]
                  for op, name in ((0, "ds_read_b128"), (1, "ds_read_b64_tr_b16"), (2, "ds_write_b128"))}
    res["copy_to_lds"] = [copy_rate(wg_per_cu=n) for n in (1, 2, 4)]
    res["mfma_valu_overlap"] = mix_rates()
    return res


def _bytes_per_clock(clocks, grid, bytes_per_wg, wall_s):
    """Bytes per shader-clock cycle per CU, grid / 256 workgroups per CU each
    moving bytes_per_wg: over the slowest workgroup's loop cycles, and over
    the launch's wall time (events) at the workgroups' average clock (shader
    cycles over 100 MHz reference ticks), which also counts the launch."""
    c = clocks.view(grid, 2).cpu().double()
    per_cu = (grid / 256) * bytes_per_wg
    ghz = float((c[:, 0] / (c[:, 1] / 100e6)).mean())
    return {"loop": round(per_cu / float(c[:, 0].max()), 1),
            "wall": round(per_cu / (wall_s * ghz), 1)}


def _timed(launch):
    import torch
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    launch()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / 1e3


def lds_rate(op, iters=20000, waves_per_cu=16):
    """LDS rate per CU (steel_lds_rate: op 0 ds_read_b128, 1 two
    ds_read_b64_tr_b16, 2 ds_write_b128, 16 bytes per lane eight times per
    iteration) with waves_per_cu waves resident on every CU (256 workgroups)."""
    import torch
    from paper_2607_09385_amd import _lib
    lib = _lib.load()
    dev = torch.device("cuda:0")
    grid = 256
    sink = torch.empty(grid * 64 * waves_per_cu, dtype=torch.int32, device=dev)
    clocks = torch.zeros(2 * grid, dtype=torch.int64, device=dev)
    stream = torch.cuda.current_stream()
    def launch(n=iters):
        st = lib.steel_lds_rate(op, n, grid, waves_per_cu, sink.data_ptr(), clocks.data_ptr(),
                                stream.cuda_stream)
        if st != 0:
            raise RuntimeError(f"steel_lds_rate failed ({st})")
    launch(iters // 4)
    wall = _timed(launch)
    return {"waves_per_cu": waves_per_cu,
            "bytes_per_clock_per_cu": _bytes_per_clock(clocks, grid, waves_per_cu * 64 * 16 * 8 * iters,
                                                       wall)}


def copy_rate(iters=1500, wg_per_cu=2, waves_per_wg=4):
    """Global -> LDS copy rate per CU (steel_copy_rate: global_load_lds_dwordx4
    filling a 32 KiB buffer per workgroup, waiting for each fill) from a 16 MiB
    source the L2s hold, with wg_per_cu workgroups of waves_per_wg waves on
    every CU."""
    import torch
    from paper_2607_09385_amd import _lib
    lib = _lib.load()
    dev = torch.device("cuda:0")
    grid = 256 * wg_per_cu
    src = torch.ones(16 << 20, dtype=torch.uint8, device=dev)
    sink = torch.empty(grid * 64 * waves_per_wg, dtype=torch.int32, device=dev)
    clocks = torch.zeros(2 * grid, dtype=torch.int64, device=dev)
    stream = torch.cuda.current_stream()
    def launch(n=iters):
        st = lib.steel_copy_rate(src.data_ptr(), src.numel(), n, grid, waves_per_wg, sink.data_ptr(),
                                 clocks.data_ptr(), stream.cuda_stream)
        if st != 0:
            raise RuntimeError(f"steel_copy_rate failed ({st})")
    launch(iters // 4)
    wall = _timed(launch)
    return {"workgroups_per_cu": wg_per_cu, "waves_per_wg": waves_per_wg,
            "bytes_per_clock_per_cu": _bytes_per_clock(clocks, grid, 32768 * iters, wall)}


def valu_rate(op, iters=200000, waves_per_wg=16, grid=256):
    """Cycles per 64-lane instruction on one SIMD (steel_valu_rate: eight
    independent chains of v_exp_f32 (op 0) or v_fma_f32 (op 1) per lane, grid *
    waves_per_wg / 1024 waves per SIMD, all resident at once), from the
    kernel's own shader-clock cycles, so independent of the clock.  With one
    wave per SIMD it is the issue interval of a single wave; with several, the
    SIMD's throughput."""
    import torch
    from paper_2607_09385_amd import _lib
    lib = _lib.load()
    dev = torch.device("cuda:0")
    seed = torch.linspace(-1.0, 1.0, 8, dtype=torch.float32, device=dev)
    sink = torch.empty(grid * 64 * waves_per_wg, dtype=torch.float32, device=dev)
    clocks = torch.zeros(2 * grid, dtype=torch.int64, device=dev)
    stream = torch.cuda.current_stream()
    for n in (iters // 4, iters):
        st = lib.steel_valu_rate(op, seed.data_ptr(), n, grid, waves_per_wg, sink.data_ptr(),
                                 clocks.data_ptr(), stream.cuda_stream)
        if st != 0:
            raise RuntimeError(f"steel_valu_rate failed ({st})")
    torch.cuda.synchronize()
    c = clocks.view(grid, 2).cpu().double()
    waves_per_simd = grid * waves_per_wg / 1024
    per_instr = float(c[:, 0].mean()) / (iters * 8 * waves_per_simd)
    return {"waves_per_simd": waves_per_simd, "cycles_per_wave_instruction": round(per_instr, 2),
            "finite": bool(torch.isfinite(sink).all().item())}


def mix_rates(mfma_iters=2000, valu_iters=1000):
    """Overlap of one wave's matrix-core work and another wave's VALU work on
    the same SIMD (steel_mix_rate: one workgroup of eight waves per CU, waves
    w and w + 4 on SIMD w % 4; waves 0-3 issue v_mfma_f32_32x32x16_bf16 on
    N(0,1) operands, waves 4-7 eight independent v_exp_f32 or v_fma_f32
    chains).  Per role: shader-clock cycles per instruction of its own loop,
    and its average clock; with both roles on, unchanged MFMA cycles mean the
    VALU work ran beside the matrix core instead of taking turns with it."""
    import torch
    from paper_2607_09385_amd import _lib
    lib = _lib.load()
    dev = torch.device("cuda:0")
    grid = 256
    g = torch.Generator().manual_seed(0)
    ops = torch.randn((8, 64, 8), generator=g).to(torch.bfloat16).to(dev)
    seed = torch.linspace(0.2, 0.9, 8, dtype=torch.float32, device=dev)
    sink = torch.empty(grid * 512, dtype=torch.float32, device=dev)
    clocks = torch.zeros(2 * 8 * grid, dtype=torch.int64, device=dev)
    stream = torch.cuda.current_stream()
    out = {"mfma_per_wave": mfma_iters * 4, "valu_per_wave": valu_iters * 8}
    for name, mode, vop in (("mfma", 1, 0), ("exp", 2, 0), ("mfma+exp", 3, 0), ("fma", 2, 1),
                            ("mfma+fma", 3, 1)):
        for _ in range(2):   # the first launch ramps the clock
            st = lib.steel_mix_rate(mode, vop, ops.data_ptr(), mfma_iters, seed.data_ptr(), valu_iters,
                                    grid, sink.data_ptr(), clocks.data_ptr(), stream.cuda_stream)
            if st != 0:
                raise RuntimeError(f"steel_mix_rate failed ({st})")
        torch.cuda.synchronize()
        c = clocks.view(grid, 8, 2).cpu().double()
        row = {}
        if mode & 1:
            m = c[:, :4]
            row["mfma_cycles"] = round(float(m[..., 0].mean()) / (mfma_iters * 4), 2)
            row["mfma_clock_ghz"] = round(float((m[..., 0] / (m[..., 1] / 100e6)).mean() / 1e9), 3)
        if mode & 2:
            v = c[:, 4:]
            row["valu_cycles"] = round(float(v[..., 0].mean()) / (valu_iters * 8), 2)
            row["valu_clock_ghz"] = round(float((v[..., 0] / (v[..., 1] / 100e6)).mean() / 1e9), 3)
        out[name] = row
    return out


COPY_BYTES = 256 << 20   # reference elementwise kernel for the counter scale


def traffic_run(name, runs):
    """Workload for the rocprofv3 counter passes: the attention run of one
    plan ``runs`` times, then one float32 elementwise kernel that reads and
    writes exactly COPY_BYTES each (its counter readings give the scale from
    counter KiB to bytes)."""
    import torch
    import workloads
    import paper_2607_09385_amd as steel

    steel.load()
    cfg = workloads.CONFIGS[name]
    q, k, v, mask = workloads.make_workload(cfg)
    dev = torch.device("cuda:0")
    qd, kd, vd = q.to(dev), k.to(dev), v.to(dev)
    md = None if mask is None else torch.from_numpy(mask).to(dev)
    out = torch.empty((cfg.B, cfg.Hq, cfg.S_q, cfg.D), dtype=torch.float32, device=dev)
    plan = steel.Plan(md, cfg.B, cfg.Hq, cfg.Hkv, cfg.S_q, cfg.S_k, causal=cfg.causal, device=dev)
    for _ in range(runs):
        plan.run(qd, kd, vd, scale=cfg.scale, out=out)
    src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    torch.add(src, 1.0, out=dst)
    torch.cuda.synchronize()
    print(f"[traffic-run] {name}: {runs} attention runs, then one {COPY_BYTES} B elementwise add",
          flush=True)


def traffic_from(fetch_dir, write_dir, name):
    """Turn the two counter passes over ``--traffic-run`` into HBM bytes per
    attention run and record them in profiles/attn_traffic.json."""
    import csv

    def per_kernel(d, counter):
        vals = {}
        for r in csv.DictReader(open(os.path.join(d, "run_counter_collection.csv"))):
            if r["Counter_Name"] != counter:
                continue
            vals.setdefault(r["Kernel_Name"].split("(")[0], []).append(float(r["Counter_Value"]))
        return {k: sum(v) / len(v) for k, v in vals.items()}

    rec = {}
    for counter, d in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        k = per_kernel(d, counter)
        ref = [v for n, v in k.items() if "elementwise" in n and "add" in n]
        attn = {n: v for n, v in k.items() if "k_attn" in n}
        scale = COPY_BYTES / (ref[0] * 1024.0)
        rec[counter] = {"scale": scale,
                        "kernels": {n: v * 1024.0 * scale for n, v in attn.items()}}
    kernels = sorted(rec["FETCH_SIZE"]["kernels"])
    per_run = sum(rec["FETCH_SIZE"]["kernels"][n] + rec["WRITE_SIZE"]["kernels"].get(n, 0.0)
                  for n in kernels)
    try:
        with open(TRAFFIC_FILE) as f:
            out = json.load(f)
        if out.get("kernel_sha") != kernel_hash():
            out = {}
    except (OSError, ValueError):
        out = {}
    out["kernel_sha"] = kernel_hash()
    out.setdefault("workloads", {})[name] = {
        "bytes_per_run": per_run,
        "fetch_bytes": rec["FETCH_SIZE"]["kernels"],
        "write_bytes": rec["WRITE_SIZE"]["kernels"],
        "scale_fetch": rec["FETCH_SIZE"]["scale"],
        "scale_write": rec["WRITE_SIZE"]["scale"],
        "reference": f"float32 elementwise add reading and writing {COPY_BYTES} B",
    }
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(out, f, indent=1, sort_keys=True)
    print(json.dumps(out["workloads"][name], indent=1))


def bench_workload(name, steps, warmup, cpu_seconds, want_cpu, clock_warmup=0.5):
    import torch
    import workloads
    import paper_2607_09385_amd as steel

    steel.load()
    cfg = workloads.CONFIGS[name]
    print(f"[bench] {name}: generating inputs", file=sys.stderr, flush=True)
    q, k, v, mask = workloads.make_workload(cfg)
    dev = torch.device("cuda:0")
    qd, kd, vd = q.to(dev), k.to(dev), v.to(dev)
    md = None if mask is None else torch.from_numpy(mask).to(dev)
    out = torch.empty((cfg.B, cfg.Hq, cfg.S_q, cfg.D), dtype=torch.float32, device=dev)
    counts = live_tile_counts(mask, cfg.B, cfg.Hq, cfg.S_q, cfg.S_k, cfg.causal)
    n_live = int(counts.sum())
    f_live = 4.0 * 64 * 64 * cfg.D * n_live
    f_dense = 4.0 * cfg.B * cfg.Hq * cfg.S_q * cfg.S_k * cfg.D

    def step():
        steel.attn_fwd(qd, kd, vd, md, scale=cfg.scale, causal=cfg.causal, out=out)

    # The chip raises its clock over the first tenths of a second of load; the
    # protocol's warm-up calls take a few milliseconds, so the same call first
    # keeps the GPU busy for clock_warmup seconds (untimed).
    t_end = time.perf_counter() + clock_warmup
    while time.perf_counter() < t_end:
        for _ in range(10):
            step()
        torch.cuda.synchronize()
    print(f"[bench] {name}: warmup {warmup}, timing {steps} steps", file=sys.stderr, flush=True)
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) / steps
    # the same calls once more with an event between each two, for the median
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    ev[0].record()
    for i in range(steps):
        step()
        ev[i + 1].record()
    torch.cuda.synchronize()
    per_call = sorted(ev[i].elapsed_time(ev[i + 1]) for i in range(steps))
    median_ms = per_call[steps // 2] if steps % 2 else 0.5 * (per_call[steps // 2 - 1] + per_call[steps // 2])

    # attention kernels alone: plan once, time runs with events on their stream
    plan = steel.Plan(md, cfg.B, cfg.Hq, cfg.Hkv, cfg.S_q, cfg.S_k, causal=cfg.causal, device=dev)
    for _ in range(warmup):
        plan.run(qd, kd, vd, scale=cfg.scale, out=out)
    stream = torch.cuda.current_stream()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(steps):
        plan.run(qd, kd, vd, scale=cfg.scale, out=out)
    e1.record(stream)
    torch.cuda.synchronize()
    run_s = e0.elapsed_time(e1) / 1e3 / steps

    achieved = f_live / run_s / 1e12
    traffic = traffic_for(name)

    # window/sink workloads: the same call with the mask generated from block
    # coordinates (no mask tensor read by the index build)
    structured = None
    structured_b16 = None
    if cfg.mask == "window_sink":
        def step_w():
            steel.attn_fwd_window(qd, kd, vd, cfg.window_blocks, cfg.sink_blocks, scale=cfg.scale,
                                  causal=cfg.causal, out=out)
        for _ in range(warmup):
            step_w()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            step_w()
        torch.cuda.synchronize()
        wall_w = (time.perf_counter() - t0) / steps
        structured = {"call": "steel_attn_fwd_window", "ms_per_step": round(wall_w * 1e3, 4),
                      "effective_tflops": round(f_live / wall_w / 1e12, 2)}
        # the same call with the output in bf16 (half the output bytes)
        out16 = torch.empty((cfg.B, cfg.Hq, cfg.S_q, cfg.D), dtype=torch.bfloat16, device=dev)
        lse16 = torch.empty((cfg.B, cfg.Hq, cfg.S_q), dtype=torch.float32, device=dev)

        def step_b():
            steel.attn_fwd_lse(qd, kd, vd, md, scale=cfg.scale, causal=cfg.causal, out=out16,
                               lse=lse16, out_dtype=torch.bfloat16)
        for _ in range(warmup):
            step_b()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            step_b()
        torch.cuda.synchronize()
        wall_b = (time.perf_counter() - t0) / steps
        structured_b16 = {"call": "steel_attn_fwd_ex (bf16 output, with lse)",
                          "ms_per_step": round(wall_b * 1e3, 4),
                          "effective_tflops": round(f_live / wall_b / 1e12, 2)}
    # the fp8 forms of the same call (E4M3 operands for P V, or for both
    # products; each has its own error budget against exact attention)
    fp8 = {}
    lse32 = torch.empty((cfg.B, cfg.Hq, cfg.S_q), dtype=torch.float32, device=dev)
    for mode, flag, what in (("pv", "STEEL_FP8_PV", "P V"), ("all", "STEEL_FP8", "both products")):
        def step_f(mode=mode):
            steel.attn_fwd_lse(qd, kd, vd, md, scale=cfg.scale, causal=cfg.causal, out=out,
                               lse=lse32, fp8=mode)
        for _ in range(warmup):
            step_f()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            step_f()
        torch.cuda.synchronize()
        wall_f = (time.perf_counter() - t0) / steps
        fp8[mode] = {"call": f"steel_attn_fwd_ex ({flag}, with lse)",
                     "dtype": f"E4M3 operands for {what}, fp32 accumulation",
                     "ms_per_step": round(wall_f * 1e3, 4),
                     "effective_tflops": round(f_live / wall_f / 1e12, 2)}
    line = {
        "metric": METRIC,
        "value": round(f_live / wall / 1e12, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "clock_warmup_s": clock_warmup,
        "ms_per_step": round(wall * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {**cfg.describe(), "live_tiles": n_live, "parallelism": "single GPU"},
        "pct_peak_effective": round(100 * f_live / wall / 1e12 / PEAK_TFLOPS, 2),
        "dense_equiv_tflops": round(f_dense / wall / 1e12, 2),
        "pct_peak_dense": round(100 * f_dense / wall / 1e12 / PEAK_TFLOPS, 2),
        "peak_tflops": round(PEAK_TFLOPS, 1),
        "peak_basis": "256 CU x 2.4 GHz x 4096 bf16 flop/clk/CU",
        "ms_per_step_median": round(median_ms, 4),
        "valu_bound": valu_bound(n_live, cfg.D),
        "roofline": {
            "bound": "mfma",
            "achieved": round(achieved, 2),
            "peak": round(PEAK_TFLOPS, 1),
            "unit": "TFLOP/s",
            "frac": round(achieved / PEAK_TFLOPS, 4),
            "traffic": traffic,
            "kernel": "attention run (k_attn_ws for uniform head packs of 4 at D=128, k_attn for the other items), index prebuilt",
            "run_us": round(run_s * 1e6, 2),
            "algorithmic_flops_per_run": f_live,
        },
    }
    # top-k workloads: the mask producer that precedes the pass, on the device
    producer = None
    if cfg.mask == "topk_meanpool":
        mask_dev = torch.empty((cfg.B, cfg.Hq, cfg.nQB, cfg.nKB), dtype=torch.uint8, device=dev)

        def step_m():
            steel.topk_block_mask(qd, kd, 1, 10, causal=cfg.causal, out=mask_dev)
        for _ in range(warmup):
            step_m()
        e0.record(stream)
        for _ in range(steps):
            step_m()
        e1.record(stream)
        torch.cuda.synchronize()
        t_m = e0.elapsed_time(e1) / 1e3 / steps
        same = bool(torch.equal(mask_dev.cpu(), torch.from_numpy(mask)))
        # algorithmic bytes: Q and K read once, the mask written once
        nbytes = 2 * (q.numel() + k.numel()) + mask_dev.numel()
        producer = {"call": "steel_topk_block_mask", "us": round(t_m * 1e6, 2),
                    "equals_workload_mask": same,
                    "roofline": {"bound": "hbm", "achieved": round(nbytes / t_m / 1e9, 1),
                                 "peak": 8000.0, "unit": "GB/s",
                                 "frac": round(nbytes / t_m / 1e9 / 8000.0, 4),
                                 "algorithmic_bytes": nbytes}}
    line["fp8"] = fp8
    if structured is not None:
        line["structured_mask"] = structured
    if structured_b16 is not None:
        line["bf16_output"] = structured_b16
    if producer is not None:
        line["mask_producer"] = producer
    if want_cpu:
        print(f"[bench] {name}: CPU oracle baseline (~{cpu_seconds}s)", file=sys.stderr, flush=True)
        line["cpu_baseline"] = cpu_baseline(cfg, q, k, v, mask, counts, cpu_seconds)
    return line


def unfused_attention(qd, kd, vd, hidden, scale):
    """Layer-by-layer attention on the same GPU (the comparison of Section V-B:
    every stage writes its result to HBM and the next reads it back):
    S = scale * Q K^T (hipBLASLt bf16 GEMM, materialised), masked with -inf,
    P = softmax(S) (materialised, bf16), O = P V (hipBLASLt).  ``hidden`` is the
    element mask of the scores that are not visible (bool [B, Hq, S_q, S_k])."""
    import torch
    B, Hq, S_q, D = qd.shape
    Hkv, S_k = kd.shape[1], kd.shape[2]
    G = Hq // Hkv
    q3 = qd.reshape(B * Hkv, G * S_q, D)
    kt = kd.reshape(B * Hkv, S_k, D).transpose(1, 2).contiguous()
    a = torch.empty((B * Hkv, G * S_q, S_k), dtype=torch.bfloat16, device=qd.device)
    torch.baddbmm(a, q3, kt, beta=0.0, alpha=scale, out=a)
    a = a.view(B, Hq, S_q, S_k).masked_fill_(hidden, float("-inf"))
    p = torch.softmax(a, dim=-1)
    o = torch.bmm(p.view(B * Hkv, G * S_q, S_k), vd.reshape(B * Hkv, S_k, D))
    return o.view(B, Hq, S_q, D)


def hidden_scores(md, B, Hq, S_q, S_k, causal, dev):
    """bool [B, Hq, S_q, S_k]: True where the block mask or the causal
    structure hides the score."""
    import torch
    if md is None:
        vis = torch.ones((B, Hq, S_q, S_k), dtype=torch.bool, device=dev)
    else:
        vis = md.bool().repeat_interleave(64, 2).repeat_interleave(64, 3)[:, :, :S_q, :S_k]
    if causal:
        vis = vis & torch.ones((S_q, S_k), dtype=torch.bool, device=dev).tril(diagonal=S_k - S_q)
    return (~vis).contiguous()


def bench_unfused(name, steps, warmup):
    """One JSON line: the layer-by-layer baseline against the fused call on
    the same workload and GPU, with the HBM bytes each moves by construction."""
    import torch
    import workloads
    import paper_2607_09385_amd as steel

    steel.load()
    cfg = workloads.CONFIGS[name]
    q, k, v, mask = workloads.make_workload(cfg)
    dev = torch.device("cuda:0")
    qd, kd, vd = q.to(dev), k.to(dev), v.to(dev)
    md = None if mask is None else torch.from_numpy(mask).to(dev)
    hidden = hidden_scores(md, cfg.B, cfg.Hq, cfg.S_q, cfg.S_k, cfg.causal, dev)
    counts = live_tile_counts(mask, cfg.B, cfg.Hq, cfg.S_q, cfg.S_k, cfg.causal)
    f_live = 4.0 * 64 * 64 * cfg.D * int(counts.sum())
    out = torch.empty((cfg.B, cfg.Hq, cfg.S_q, cfg.D), dtype=torch.float32, device=dev)

    def timed(fn, n_warm, n):
        for _ in range(n_warm):
            fn()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(n):
            fn()
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) / n

    t_unf = timed(lambda: unfused_attention(qd, kd, vd, hidden, cfg.scale), warmup, steps)
    t_fus = timed(lambda: steel.attn_fwd(qd, kd, vd, md, scale=cfg.scale, causal=cfg.causal, out=out),
                  warmup, steps)
    o_unf = unfused_attention(qd, kd, vd, hidden, cfg.scale).float()
    steel.attn_fwd(qd, kd, vd, md, scale=cfg.scale, causal=cfg.causal, out=out)
    torch.cuda.synchronize()
    diff = (o_unf - out).abs()
    n_sc = cfg.B * cfg.Hq * cfg.S_q * cfg.S_k
    qkv = 2 * (q.numel() + k.numel() + v.numel())
    # by construction: GEMM writes S (2 B/score); the mask pass reads S and the
    # mask and writes S (5 B); softmax reads S, writes P (4 B); the PV GEMM
    # reads P (2 B); plus Q, K, V read and O written (bf16)
    unf_bytes = qkv + 13 * n_sc + 2 * q.numel()
    fus_bytes = qkv + 4 * q.numel() + (0 if mask is None else mask.size)
    return {
        "baseline": "layer-by-layer attention (hipBLASLt GEMMs, softmax and mask passes, scores and P materialised in bf16)",
        "workload": name,
        "unfused_ms": round(t_unf * 1e3, 3),
        "fused_ms": round(t_fus * 1e3, 3),
        "speedup_fused": round(t_unf / t_fus, 2),
        "unfused_effective_tflops": round(f_live / t_unf / 1e12, 2),
        "fused_effective_tflops": round(f_live / t_fus / 1e12, 2),
        "hbm_bytes_model": {"unfused": unf_bytes, "fused_algorithmic": fus_bytes},
        "max_abs_diff_vs_fused": float(diff.max().item()),
        "mean_abs_diff_vs_fused": float(diff.mean().item()),
        "steps": steps, "warmup": warmup,
    }


def unfused_traffic_run(name):
    """Workload for counter passes over the layer-by-layer baseline: one warm
    call, then a float32 elementwise add of COPY_BYTES, one unfused call, and
    the add again (the two adds bracket the call's dispatches and scale the
    counters)."""
    import torch
    import workloads

    cfg = workloads.CONFIGS[name]
    q, k, v, mask = workloads.make_workload(cfg)
    dev = torch.device("cuda:0")
    qd, kd, vd = q.to(dev), k.to(dev), v.to(dev)
    md = None if mask is None else torch.from_numpy(mask).to(dev)
    hidden = hidden_scores(md, cfg.B, cfg.Hq, cfg.S_q, cfg.S_k, cfg.causal, dev)
    src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    unfused_attention(qd, kd, vd, hidden, cfg.scale)
    torch.cuda.synchronize()
    torch.add(src, 1.0, out=dst)
    torch.cuda.synchronize()
    unfused_attention(qd, kd, vd, hidden, cfg.scale)
    torch.cuda.synchronize()
    torch.add(src, 1.0, out=dst)
    torch.cuda.synchronize()
    print(f"[unfused-traffic-run] {name}: one unfused call between two {COPY_BYTES} B adds", flush=True)


def unfused_traffic_from(fetch_dir, write_dir):
    """HBM bytes of the unfused call from the two counter passes over
    ``--unfused-traffic-run``: the dispatches between the last two adds."""
    import csv
    out = {}
    for counter, d in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        rows = [r for r in csv.DictReader(open(os.path.join(d, "run_counter_collection.csv")))
                if r["Counter_Name"] == counter]
        rows.sort(key=lambda r: int(r["Dispatch_Id"]))
        adds = [i for i, r in enumerate(rows) if "elementwise" in r["Kernel_Name"] and "add" in r["Kernel_Name"]]
        a, b = adds[-2], adds[-1]
        scale = COPY_BYTES / (float(rows[a]["Counter_Value"]) * 1024.0)
        between = rows[a + 1:b]
        out[counter] = {"bytes": sum(float(r["Counter_Value"]) for r in between) * 1024.0 * scale,
                        "dispatches": len(between), "scale": scale}
    out["total_bytes"] = out["FETCH_SIZE"]["bytes"] + out["WRITE_SIZE"]["bytes"]
    print(json.dumps(out, indent=1))


def bench_merge(name, parts, steps, warmup):
    """Time of steel_attn_merge over ``parts`` partial outputs of the
    workload's output shape, against the HBM roofline (each part's O and lse
    read once, O and lse written once)."""
    import torch
    import workloads
    import paper_2607_09385_amd as steel

    steel.load()
    cfg = workloads.CONFIGS[name]
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev).manual_seed(0)
    o = torch.randn((parts, cfg.B, cfg.Hq, cfg.S_q, cfg.D), generator=g, device=dev)
    l = torch.randn((parts, cfg.B, cfg.Hq, cfg.S_q), generator=g, device=dev)
    out = torch.empty(o.shape[1:], device=dev)
    lo = torch.empty(l.shape[1:], device=dev)
    for _ in range(warmup):
        steel.attn_merge(o, l, out=out, lse_out=lo)
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(steps):
        steel.attn_merge(o, l, out=out, lse_out=lo)
    e1.record(stream)
    torch.cuda.synchronize()
    t = e0.elapsed_time(e1) / 1e3 / steps
    nbytes = 4 * (o.numel() + l.numel() + out.numel() + lo.numel())
    return {"call": "steel_attn_merge", "workload_shape": name, "parts": parts,
            "us": round(t * 1e6, 2),
            "roofline": {"bound": "hbm", "achieved": round(nbytes / t / 1e9, 1), "peak": HBM_PEAK_GBS,
                         "unit": "GB/s", "frac": round(nbytes / t / 1e9 / HBM_PEAK_GBS, 4),
                         "algorithmic_bytes": nbytes}}


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=25)
    ap.add_argument("--clock-warmup", type=float, default=0.5,
                    help="seconds of untimed calls before the warm-up steps (clock ramp)")
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--all", action="store_true", help="one line per named workload")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--traffic-run", action="store_true",
                    help="workload for the rocprofv3 FETCH_SIZE / WRITE_SIZE passes")
    ap.add_argument("--traffic-from", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="record HBM bytes per run from the two counter passes")
    ap.add_argument("--unfused", action="store_true",
                    help="layer-by-layer baseline against the fused call (one JSON line)")
    ap.add_argument("--merge", type=int, default=0, metavar="PARTS",
                    help="time steel_attn_merge over PARTS partial outputs of the workload's shape")
    ap.add_argument("--mfma-peak", action="store_true",
                    help="achievable bf16 MFMA rate for constant and N(0,1) operands (one JSON line)")
    ap.add_argument("--unfused-traffic-run", action="store_true",
                    help="workload for counter passes over the layer-by-layer baseline")
    ap.add_argument("--unfused-traffic-from", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="HBM bytes of one layer-by-layer call from the two counter passes")
    args = ap.parse_args()
    if args.unfused_traffic_from:
        unfused_traffic_from(*args.unfused_traffic_from)
        return
    if args.traffic_from:
        traffic_from(args.traffic_from[0], args.traffic_from[1], args.workload)
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py: measures one GPU only (asked for --gpus {args.gpus}, "
              f"WORLD_SIZE={world}); the path would shard by key/value group with no "
              "exchange between GPUs, which is not implemented", file=sys.stderr)
        sys.exit(2)
    if args.traffic_run:
        traffic_run(args.workload, args.steps if args.steps != 50 else 5)
        return
    if args.mfma_peak:
        print(json.dumps({"mfma_peak": mfma_peak(), "peak_tflops": round(PEAK_TFLOPS, 1)}), flush=True)
        return
    if args.merge:
        print(json.dumps(bench_merge(args.workload, args.merge, args.steps, args.warmup)), flush=True)
        return
    if args.unfused_traffic_run:
        unfused_traffic_run(args.workload)
        return
    if args.unfused:
        print(json.dumps(bench_unfused(args.workload, args.steps if args.steps != 50 else 10,
                                       args.warmup if args.warmup != 25 else 3)), flush=True)
        return
    import workloads
    names = workloads.CONFIG_ORDER if args.all else [args.workload]
    for i, name in enumerate(names):
        want_cpu = (not args.no_cpu_baseline) and (name == args.workload or not args.all)
        line = bench_workload(name, args.steps, args.warmup, args.cpu_seconds, want_cpu,
                              args.clock_warmup)
        print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
