#!/usr/bin/env python3
"""Benchmark of the COVER hot path on one MI355X.

A step is one pass of the whole hot path for one layer of a decoding step at the
LLaDA-8B layer shape (B=1, H=32, L=1024 = 768 prompt + 256 generated, d=128, bf16):
  cover_attn_fwd      KV-cache-override attention with the diagonal correction (16 seeds)
  cover_select_seeds  stability-aware scores, adaptive budget, top-k over the 256 generated
                      positions
on seeded synthetic inputs already resident in HBM.  Prints one JSON line.

  python bench.py [--steps K] [--warmup W] [--workload llada|dream|batched] [--settle-ms T]

Before the W warm-up steps, the timed operation runs back to back, untimed, for T ms of wall
time (default 100; 0 turns it off).  The GPU raises its clocks over the first tens of
milliseconds of sustained load: on an MI355X the layer step takes about 31 us in the first
6 ms and settles at about 27.5 us after about 25 ms.  A decoding loop runs in the settled
state, so that is the state the timed steps measure.

Profiling helpers (what the committed rocprofv3 summaries were made with):
  --only attn|select   time only that kernel in the step
  --copy-mib N         run a plain device copy of N MiB (HBM counter calibration)
  --kernel token_stats|attn_stats
                       time one producer of the selection inputs at the LLaDA-8B step shape
                       (the LM head's 256 x 126464 bf16 logits; the 256-position generated
                       block of the last layer) and print its own JSON line
  --workload step      the full decode step of a random-init 32-layer LLaDA-8B-shaped model
                       (torch for the rest of the model, this library for every layer's
                       attention, the token statistics, attention masses and seed selection);
                       prints its own JSON line with the attention share of the step
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6   # 256 CU x 4096 dense bf16 flop/clk x 2.4 GHz
PEAK_HBM_GBS = 8000.0
KERNEL_SOURCES = ("paper_2602_06161_amd/csrc/cover_attn_w4.hip",)
TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "attn_{workload}_hbm_traffic.md")


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(workload: str):
    """HBM bytes per attention launch from the committed rocprofv3 counter summary of this
    workload, if it was taken on the current kernel source; else None."""
    path = TRAFFIC_SUMMARY.format(workload=workload)
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m = re.search(r"^traffic_bytes_per_launch:\s*(\d+)\s+workload:\s*(\w+)\s+source:\s*(\w+)",
                  text, flags=re.M)
    if not m or m.group(2) != workload or m.group(3) != kernel_source_hash():
        return None
    return int(m.group(1))


def settle_clocks(fn, ms: float, sync=None) -> int:
    """Run `fn` back to back for `ms` milliseconds of wall time, untimed, so that the timed
    launches see the clocks of sustained load; returns how many calls it made.  `sync` waits
    for the queued work (the device by default), every 16 calls."""
    if sync is None:
        import torch

        sync = torch.cuda.synchronize
    n = 0
    t_end = time.perf_counter() + ms * 1e-3
    while time.perf_counter() < t_end:
        for _ in range(16):
            fn()
        sync()
        n += 16
    return n


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--settle-ms", type=float, default=100.0,
                    help="untimed back-to-back run before the warm-up steps (clock ramp)")
    ap.add_argument("--ramp-windows", type=int, default=0,
                    help="first time N consecutive windows of 200 steps (the clock ramp) and "
                         "report them as ramp_us_per_step")
    ap.add_argument("--workload", default="llada", choices=["llada", "dream", "batched", "step", "loop", "block"])
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--only", choices=["attn", "select"], default=None)
    ap.add_argument("--copy-mib", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-phase-timing", action="store_true",
                    help="skip the shader-clock / phase leg (a child process running the timing "
                         "build of the attention kernel once)")
    ap.add_argument("--calibrate-mfma", action="store_true",
                    help="run the pure-MFMA calibration kernel of the timing build (one "
                         "workgroup of four waves per CU, bf16 32x32x16 MFMAs only) K times; "
                         "the reference for the MFMA counters")
    ap.add_argument("--phase-timing", action="store_true",
                    help="run the attention kernel of the timing build of the library "
                         "(lib/libcover_timing.so) once after warm-up and print where a "
                         "workgroup's cycles go, and the shader clock under load (with "
                         "--workload block: the single-launch block attention kernel)")
    ap.add_argument("--zero-seeds", action="store_true",
                    help="with --phase-timing: the same attention launch with empty seed lists")
    ap.add_argument("--kernel", choices=["token_stats", "token_sample", "attn_stats",
                                         "decode_update"], default=None)
    ap.add_argument("--lm-scale", type=float, default=8.0,
                    help="loop workload: LM-head weights scaled by this (peaked distributions)")
    ap.add_argument("--max-steps", type=int, default=2048, help="loop workload: step budget")
    ap.add_argument("--tau", type=float, default=0.9, help="loop workload: drafting threshold")
    ap.add_argument("--remask-budget", type=int, default=5,
                    help="loop workload: ReMasks after which a position is no longer a seed")
    ap.add_argument("--temperature", type=float, default=0.0,
                    help="loop workload: sampling temperature of the predictions (0 = argmax)")
    ap.add_argument("--min-draft", type=int, default=1,
                    help="loop workload: draft at least this many per step (0 = the paper's rule)")
    ap.add_argument("--block-len", type=int, default=64,
                    help="loop workload: semi-autoregressive block length (Sec. 6.1: 64 for LLaDA)")
    ap.add_argument("--variant", choices=["cover", "wo_kv", "wo_seed"], default="cover",
                    help="loop workload: COVER, or the ablations of Sec. 6.4 (no KV override; "
                         "confidence-drop seeds)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py: measures a single GPU only (the path is not sharded across GPUs). "
              "Run with --gpus 1.", file=sys.stderr)
        return 2

    import torch
    from paper_2602_06161_amd import cover, synth

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)

    if args.copy_mib:
        n = args.copy_mib * (1 << 20) // 4
        src = torch.ones(n, device=dev, dtype=torch.float32)
        dst = torch.empty_like(src)
        for _ in range(args.steps):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_mib": args.copy_mib, "launches": args.steps}))
        return 0

    if args.phase_timing:
        if args.workload == "block":
            return bench_block_phase_timing(args, dev, stream)
        return bench_phase_timing(args, dev, stream)
    if args.calibrate_mfma:
        return bench_calibrate_mfma(args, dev, stream)
    if args.kernel:
        return bench_producer(args, dev, stream)
    if args.workload == "block":
        return bench_block(args, dev, stream)
    if args.workload in ("step", "loop"):
        return bench_full_step(args, dev, stream, loop=args.workload == "loop")

    a = synth.step_inputs(args.workload, seed=args.seed)
    c = a["cfg"]
    t = {k: a[k].to(dev) for k in ("q", "k_live", "v_live", "k_cache", "v_cache", "seed_idx",
                                   "n_seed", "logp", "d_in", "d_out", "flags")}
    out = torch.empty_like(t["q"])
    lse = torch.empty((c.B, c.Hq, c.L), device=dev, dtype=torch.float32)
    max_seeds = c.n_seeds
    nsi = torch.empty((c.B, max_seeds), device=dev, dtype=torch.int32)
    nns = torch.empty((c.B,), device=dev, dtype=torch.int32)
    score = torch.empty((c.B, a["Lr"]), device=dev, dtype=torch.float64)

    # arguments marshalled once, so the timed loop is not bound by Python launch overhead
    attn = cover.PreparedAttn(t["q"], t["k_live"], t["v_live"], t["k_cache"], t["v_cache"],
                              t["seed_idx"], t["n_seed"], out=out, lse=lse, stream=stream)
    select = cover.PreparedSelect(t["logp"], t["d_in"], t["d_out"], t["flags"], max_seeds,
                                  a["pos_offset"], seed_idx=nsi, n_seed=nns, score=score,
                                  stream=stream)

    do_attn = args.only in (None, "attn")
    do_sel = args.only in (None, "select")

    def one_step():
        if do_attn:
            attn()
        if do_sel:
            select()

    ramp = []
    for _ in range(args.ramp_windows):  # the clock ramp, window by window, from a cold start
        r0, r1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        r0.record(stream)
        for _ in range(200):
            one_step()
        r1.record(stream)
        torch.cuda.synchronize()
        ramp.append(round(r0.elapsed_time(r1) * 1e3 / 200, 3))
    settle_clocks(one_step, args.settle_ms)
    for _ in range(args.warmup):
        if do_attn:
            attn()
        if do_sel:
            select()
    torch.cuda.synchronize()

    K = args.steps
    ev_step0 = torch.cuda.Event(enable_timing=True)
    ev_step1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev_step0.record(stream)
    for _ in range(K):
        if do_attn:
            attn()
        if do_sel:
            select()
    ev_step1.record(stream)
    torch.cuda.synchronize()
    t1 = time.perf_counter()

    wall_ms = (t1 - t0) * 1e3 / K
    gpu_ms = ev_step0.elapsed_time(ev_step1) / K
    ms_per_step = max(wall_ms, gpu_ms)
    flops = cover.attn_flops(c.B, c.Hq, c.L, c.d)

    # Roofline leg: the attention kernel alone, K launches back to back on the same stream,
    # bracketed by events (its average launch duration, as a kernel trace reports it).
    attn_us = None
    if do_attn:
        ea0 = torch.cuda.Event(enable_timing=True)
        ea1 = torch.cuda.Event(enable_timing=True)
        ea0.record(stream)
        for _ in range(K):
            attn()
        ea1.record(stream)
        torch.cuda.synchronize()
        attn_us = ea0.elapsed_time(ea1) * 1e3 / K

    # Cold leg: the same launches rotating over copies of the inputs and outputs at other
    # addresses, more than 256 MiB in all, so that no launch finds its operands in the
    # last-level (Infinity) cache left by the previous one.
    attn_cold_us, cold_sets = None, 0
    if do_attn and not args.only:
        names = ("q", "k_live", "v_live", "k_cache", "v_cache")
        set_bytes = sum(t[k].numel() * t[k].element_size() for k in names) + out.numel() * out.element_size()
        cold_sets = max(2, -(-(320 << 20) // set_bytes))
        sets = []
        for _ in range(cold_sets):
            cp = {k: t[k].clone() for k in names}
            sets.append(cover.PreparedAttn(cp["q"], cp["k_live"], cp["v_live"], cp["k_cache"],
                                           cp["v_cache"], t["seed_idx"], t["n_seed"],
                                           out=torch.empty_like(out), lse=lse, stream=stream))
        for s_ in sets:
            s_()
        torch.cuda.synchronize()
        ec0 = torch.cuda.Event(enable_timing=True)
        ec1 = torch.cuda.Event(enable_timing=True)
        ec0.record(stream)
        for k in range(K):
            sets[k % cold_sets]()
        ec1.record(stream)
        torch.cuda.synchronize()
        attn_cold_us = ec0.elapsed_time(ec1) * 1e3 / K
        del sets
    if args.only:
        print(json.dumps({"only": args.only, "us_per_launch": round(ms_per_step * 1e3, 3),
                          "attn_event_us": attn_us, "steps": K}))
        return 0

    value = flops / (ms_per_step * 1e-3) / 1e12
    attn_tflops = flops / (attn_us * 1e-6) / 1e12
    traffic = measured_traffic(args.workload)
    rec = {
        "metric": "COVER-attention TFLOP/s + us/layer-step at LLaDA-8B shape; % bf16 MFMA peak",
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "settle_ms": args.settle_ms,
        **({"ramp_us_per_step": ramp} if ramp else {}),
        "ms_per_step": round(ms_per_step, 5),
        "us_per_layer_step": round(ms_per_step * 1e3, 3),
        "pct_bf16_peak": round(100 * value / PEAK_BF16_TFLOPS, 2),
        "attn_kernel_us": round(attn_us, 3),
        "attn_kernel_tflops": round(attn_tflops, 2),
        "attn_kernel_pct_bf16_peak": round(100 * attn_tflops / PEAK_BF16_TFLOPS, 2),
        "attn_kernel_us_cold": None if attn_cold_us is None else round(attn_cold_us, 3),
        "cold_sets": cold_sets,
        "wall_ms_per_step": round(wall_ms, 5),
        "gpu_ms_per_step": round(gpu_ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) q/k/v/cache, Beta(5,1) confidences)",
        "config": {"workload": f"{args.workload} layer step: B={c.B} Hq={c.Hq} Hkv={c.Hkv} "
                               f"L={c.L} d={c.d} seeds={c.n_seeds}, selection Lr={a['Lr']}",
                   "B": c.B, "Hq": c.Hq, "Hkv": c.Hkv, "L": c.L, "d": c.d,
                   "n_seed": c.n_seeds, "Lr": a["Lr"], "parallelism": "single GPU"},
        "roofline": {
            "bound": "mfma",
            "kernel": "cover_attn_w4_kernel",
            "achieved": round(attn_tflops, 2),
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(attn_tflops / PEAK_BF16_TFLOPS, 4),
            "traffic": traffic,
            "algorithmic_flops_per_launch": flops,
        },
    }
    if not args.no_phase_timing:
        ph = phase_leg(args.workload, args.settle_ms)
        if ph is not None:
            rec["sclk_ghz_under_load"] = ph["sclk_ghz_median"]
            rec["phase_cycles_median"] = ph["cycles_median"]
    if not args.no_cpu_baseline:
        rec["cpu_baseline"] = cpu_baseline(a, flops)
    print(json.dumps(rec))
    return 0


def phase_leg(workload: str, settle_ms: float):
    """The timing build of the attention kernel, run once after warm-up in a child process
    (`--phase-timing`): the shader clock under load and the per-phase cycle medians.  None
    (with a note on stderr) if that run fails."""
    import subprocess

    cmd = [sys.executable, os.path.abspath(__file__), "--phase-timing", "--workload", workload,
           "--warmup", "5", "--settle-ms", str(settle_ms)]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    lines = [ln for ln in r.stdout.splitlines() if ln.startswith("{")]
    if r.returncode != 0 or not lines:
        print(f"bench.py: phase-timing leg failed (rc {r.returncode}): {r.stderr[-400:]}",
              file=sys.stderr)
        return None
    return json.loads(lines[-1])


def bench_producer(args, dev, stream) -> int:
    """One producer of the selection signals, K back-to-back launches between two events."""
    import ctypes

    import torch
    from paper_2602_06161_amd import cover, synth

    if args.kernel == "token_stats":
        R, V = 256, 126464
        t = synth.token_inputs(R, V, seed=args.seed)
        logits = t["buffer"].to(dev)[:, :V]
        tokens = t["tokens"].to(dev)
        outs = [torch.empty(R, device=dev, dtype=dt) for dt in (torch.float32, torch.float32,
                                                                 torch.int32)]
        desc = cover.TokenDesc(R, V, cover.COVER_BF16, logits.stride(0))
        cargs = [cover._ptr(logits), cover._ptr(tokens)] + [cover._ptr(o) for o in outs] + \
                [ctypes.byref(desc), cover._stream(stream)]
        fn = cover.lib().cover_token_stats
        run = lambda: fn(*cargs)  # arguments marshalled once (no Python work per launch)
        nbytes = R * V * 2 + R * 16  # logits once; token id in; logp, conf, argmax out
        cfg = {"workload": f"LLaDA-8B LM-head block: R={R} positions x V={V} bf16 logits"}
        bound, unit, peak = "hbm", "GB/s", PEAK_HBM_GBS
    elif args.kernel == "token_sample":
        R, V = 256, 126464
        t = synth.token_inputs(R, V, seed=args.seed)
        logits = t["buffer"].to(dev)[:, :V]
        tok = torch.empty(R, device=dev, dtype=torch.int32)
        prob = torch.empty(R, device=dev, dtype=torch.float32)
        desc = cover.TokenDesc(R, V, cover.COVER_BF16, logits.stride(0))
        cargs = [cover._ptr(logits), ctypes.c_float(0.3), ctypes.c_uint64(args.seed),
                 ctypes.c_uint32(1), cover._ptr(tok), cover._ptr(prob), ctypes.byref(desc),
                 cover._stream(stream)]
        fn = cover.lib().cover_token_sample
        run = lambda: fn(*cargs)
        nbytes = R * V * 2 + R * 8  # logits once; token and probability out
        cfg = {"workload": f"LLaDA-8B LM-head block: R={R} positions x V={V} bf16 logits, T=0.3"}
        bound, unit, peak = "hbm", "GB/s", PEAK_HBM_GBS
    elif args.kernel == "decode_update":
        B, Lr = 1, 256
        u = synth.update_inputs(B, Lr, seed=args.seed)
        t = {k: u[k].to(dev) for k in ("tokens", "argmax", "conf", "seed_idx", "n_seed",
                                         "remask_count")}
        outs = [torch.empty((B, Lr), device=dev, dtype=torch.uint8) for _ in range(2)] + \
               [torch.empty((B, 5), device=dev, dtype=torch.int32)]
        last = torch.full((B, Lr), -1, device=dev, dtype=torch.int32)
        ff = torch.empty(B, device=dev, dtype=torch.int32)
        desc = cover.UpdateDesc(B, Lr, t["seed_idx"].shape[1], u["pos_offset"], u["mask_id"], 15,
                                5, 0.9, 0)
        # the state changes in place each launch; the work per launch stays the same shape
        cargs = [cover._ptr(t[k]) for k in ("tokens", "argmax", "conf", "seed_idx", "n_seed",
                                            "remask_count")] + [cover._ptr(o) for o in outs] + \
                [cover._ptr(last), cover._ptr(ff), ctypes.byref(desc), cover._stream(stream)]
        fn = cover.lib().cover_decode_update
        run = lambda: fn(*cargs)
        nbytes = None
        flops = 0
        cfg = {"workload": f"LLaDA-8B generated block: B={B} Lr={Lr}, 16 seeds, cap 15"}
        bound, unit, peak = "latency", "us", None
    else:
        a = synth.stats_inputs("llada", seed=args.seed)
        t = {k: a[k].to(dev) for k in ("q", "k_live", "v_live", "k_cache", "v_cache", "seed_idx",
                                         "n_seed", "masked", "drafted")}
        _, lse = cover.cover_attn_fwd(t["q"], t["k_live"], t["v_live"], t["k_cache"], t["v_cache"],
                                      t["seed_idx"], t["n_seed"], stream=stream)
        c = a["cfg"]
        ws = torch.empty(cover.attn_stats_workspace(c.B, c.Hq, a["Lr"]), device=dev,
                         dtype=torch.float32)
        d_in = torch.empty((c.B, a["Lr"]), device=dev, dtype=torch.float32)
        d_out = torch.empty_like(d_in)
        desc = cover.StatsDesc(cover.attn_desc(t["q"], t["k_live"], t["seed_idx"].shape[-1]),
                               a["r0"], a["Lr"])
        cargs = [cover._ptr(x) for x in (t["q"], t["k_live"], t["k_cache"], t["seed_idx"],
                                         t["n_seed"], lse, t["masked"], t["drafted"], d_in, d_out,
                                         ws)] + [ctypes.byref(desc), cover._stream(stream)]
        fn = cover.lib().cover_attn_stats
        run = lambda: fn(*cargs)
        nbytes = None
        flops = 2 * c.B * c.Hq * a["Lr"] * a["Lr"] * c.d  # one QK^T over the region
        cfg = {"workload": f"LLaDA-8B last layer, generated block: B={c.B} Hq={c.Hq} "
                           f"Lr={a['Lr']} of L={c.L}, d={c.d} bf16"}
        bound, unit, peak = "latency", "TFLOP/s", PEAK_BF16_TFLOPS
    settle_clocks(run, args.settle_ms)
    for _ in range(args.warmup):
        if run() != 0:
            raise RuntimeError(f"{args.kernel} launch rejected")
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        run()
    e1.record(stream)
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / args.steps
    if nbytes is not None:
        achieved = nbytes / (us * 1e-6) / 1e9
    elif peak is not None:
        achieved = flops / (us * 1e-6) / 1e12
    else:  # latency-bound with no meaningful rate: the launch time itself
        achieved = us
    print(json.dumps({"kernel": args.kernel, "us_per_launch": round(us, 3), "steps": args.steps,
                      "config": cfg, "roofline": {"bound": bound, "achieved": round(achieved, 2),
                      "peak": peak, "unit": unit,
                      "frac": round(achieved / peak, 4) if peak else None,
                      "algorithmic_bytes_per_launch": nbytes}}))
    return 0


def bench_full_step(args, dev, stream, loop: bool = False) -> int:
    """The full decode step of a random-init LLaDA-8B-shaped model (32 layers, hidden 4096, 32
    heads of 128, SwiGLU FFN 12288, RMSNorm, RoPE, vocabulary 126464; B=1, L=1024 = 768 prompt +
    256 generated, bf16): torch GEMMs and element-wise ops for the rest of the model, the COVER
    library for every layer's attention (each layer's cache = its K/V buffer of the previous
    step), then LM head on the generated block, token statistics, the decoding-state update
    (drafting, revision, flags), the last layer's attention masses and the seed selection.  Prints its own JSON line with the attention share."""
    import numpy as np
    import torch
    from paper_2602_06161_amd import cover

    n_layers, H, d, hidden, ffn, vocab = 32, 32, 128, 4096, 12288, 126464
    L, prompt, gen, n_unmasked, n_seeds, max_seeds, cap = 1024, 768, 256, 128, 16, 16, 15
    mask_id = vocab - 1
    g = torch.Generator(device=dev)
    g.manual_seed(args.seed)
    w = lambda *shape: torch.randn(*shape, device=dev, dtype=torch.bfloat16, generator=g) * 0.02
    emb, lm_head = w(vocab, hidden), w(hidden, vocab)
    layers = [dict(wqkv=w(hidden, 3 * hidden), wo=w(hidden, hidden), wgu=w(hidden, 2 * ffn),
                   wd=w(ffn, hidden)) for _ in range(n_layers)]
    # per-layer K/V buffers, [L, H, d]; the previous step's buffer is this step's cache
    kv = [[(torch.zeros(L, H, d, device=dev, dtype=torch.bfloat16),
            torch.zeros(L, H, d, device=dev, dtype=torch.bfloat16)) for _ in range(n_layers)]
          for _ in range(2)]
    inv = 1.0 / (10000.0 ** (torch.arange(0, d, 2, device=dev, dtype=torch.float32) / d))
    ang = torch.arange(L, device=dev, dtype=torch.float32)[:, None] * inv[None, :]
    cos, sin = ang.cos()[:, None, :], ang.sin()[:, None, :]

    # decoding state: the 768-token prompt, 128 of the 256 generated positions unmasked, 16
    # seeds among those (fed as [MASK] for verification, Sec. 5.1)
    rng = np.random.default_rng(args.seed)
    tokens = rng.integers(0, vocab - 1, size=L)
    unm = prompt + np.sort(rng.choice(gen, n_unmasked, replace=False))
    seeds = np.sort(rng.choice(unm, n_seeds, replace=False))
    masked = np.ones(gen, np.uint8)
    masked[unm - prompt] = 0
    inp = tokens.copy()
    inp[prompt:][masked == 1] = mask_id
    inp[seeds] = mask_id
    ids = torch.from_numpy(inp).to(dev)
    # the region's state before the step (each timed step starts from it again)
    tok0 = torch.from_numpy(np.where(masked == 1, mask_id, tokens[prompt:]).astype(np.int32))
    tok0 = tok0[None].to(dev)
    cnt0 = torch.zeros((1, gen), dtype=torch.int32, device=dev)
    seed_idx = torch.from_numpy(seeds.astype(np.int32))[None].to(dev)
    n_seed = torch.tensor([n_seeds], dtype=torch.int32, device=dev)

    def rmsnorm(x):
        xf = x.float()
        return (xf * torch.rsqrt(xf.pow(2).mean(-1, keepdim=True) + 1e-6)).to(torch.bfloat16)

    def rope(x):  # [L, H, d]
        xf = x.float()
        a, b = xf[..., : d // 2], xf[..., d // 2:]
        return torch.cat((a * cos - b * sin, b * cos + a * sin), -1).to(torch.bfloat16)

    as4 = lambda t: t.unsqueeze(0).permute(0, 2, 1, 3)  # [L, H, d] -> [1, H, L, d] view
    attn_ev = []

    def model(ids, parity: int, seed_idx, n_seed, timed: bool):
        """The 32 layers on input ids; layer li's K/V go to kv[parity][li], its cache is
        kv[1 - parity][li].  Returns the generated block's logits, the last layer's lse and q."""
        x = emb[ids]
        lse = q_last = None
        for li, ly in enumerate(layers):
            h = rmsnorm(x)
            qkv = (h @ ly["wqkv"]).view(L, 3, H, d)
            q = rope(qkv[:, 0])
            k_cur, v_cur = kv[parity][li]
            k_prev, v_prev = kv[1 - parity][li]
            k_cur.copy_(rope(qkv[:, 1]))
            v_cur.copy_(qkv[:, 2])
            o = torch.empty_like(q)
            if timed:
                e = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                e[0].record(stream)
            _, lse = cover.cover_attn_fwd(as4(q), as4(k_cur), as4(v_cur), as4(k_prev), as4(v_prev),
                                          seed_idx, n_seed, out=as4(o), stream=stream,
                                          want_lse=li == n_layers - 1)
            if timed:
                e[1].record(stream)
                attn_ev.append(e)
            x = x + o.view(L, hidden) @ ly["wo"]
            gu = rmsnorm(x) @ ly["wgu"]
            x = x + (torch.nn.functional.silu(gu[:, :ffn]) * gu[:, ffn:]) @ ly["wd"]
            q_last = q
        return rmsnorm(x[prompt:]) @ lm_head, lse, q_last              # [256, vocab]

    if loop:
        return decode_loop(args, dev, stream, model, emb, lm_head, kv, as4, tokens, L, prompt, gen,
                           mask_id, max_seeds, cap, n_layers)

    def step(parity: int, timed: bool):
        logits, lse, q_last = model(ids, parity, seed_idx, n_seed, timed)
        _, conf, am = cover.cover_token_stats(logits, want_logp=False, stream=stream)
        # drafting (at most 15 above 0.9), revision of the seeds, state update, flags
        tok_state, cnt_state = tok0.clone(), cnt0.clone()
        flags, drafted, _ = cover.cover_decode_update(tok_state, am[None], conf[None], seed_idx,
                                                      n_seed, cnt_state, mask_id, 0.9, cap, 5,
                                                      prompt, stream=stream)
        # u(j) of the tokens now in place (Sec. 5.3)
        logp, _, _ = cover.cover_token_stats(logits, tok_state[0], want_conf=False,
                                             want_argmax=False, stream=stream)
        # d_in over M_t, the masked set after the update (Sec. 5.3)
        masked_now = (tok_state == mask_id).to(torch.uint8)
        k_cur, _ = kv[parity][n_layers - 1]
        k_prev, _ = kv[1 - parity][n_layers - 1]
        d_in, d_out = cover.cover_attn_stats(as4(q_last), as4(k_cur), as4(k_prev), seed_idx, n_seed,
                                             lse, masked_now, drafted, prompt, stream=stream)
        return cover.cover_select_seeds(logp[None], d_in, d_out, flags, max_seeds, prompt,
                                        stream=stream)

    for i in range(2):  # warm-up; the first fills the caches
        step(i & 1, False)
    torch.cuda.synchronize()
    K = max(1, min(args.steps, 20))
    times = []
    for i in range(K):
        attn_ev.clear()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        step(i & 1, True)
        e1.record(stream)
        torch.cuda.synchronize()
        step_ms = e0.elapsed_time(e1)
        attn_ms = sum(a.elapsed_time(b) for a, b in attn_ev)
        times.append((step_ms, attn_ms))
    times.sort()
    step_ms, attn_ms = times[len(times) // 2]
    flops_attn = n_layers * cover.attn_flops(1, H, L, d)
    flops_step = flops_attn + n_layers * 2 * L * hidden * (3 * hidden + hidden + 3 * ffn) + \
        2 * gen * hidden * vocab
    print(json.dumps({
        "workload": "full decode step, random-init LLaDA-8B-shaped model (32 layers, hidden 4096, "
                    "32 heads x 128, SwiGLU 12288, vocab 126464), B=1 L=1024 (768 + 256), 16 seeds",
        "steps": K, "step_ms": round(step_ms, 3), "attn_ms": round(attn_ms, 3),
        "attn_share": round(attn_ms / step_ms, 4),
        "attn_us_per_layer": round(attn_ms * 1e3 / n_layers, 3),
        "attn_flops_share": round(flops_attn / flops_step, 4),
        "step_tflops": round(flops_step / (step_ms * 1e-3) / 1e12, 1),
        "dtype": "bf16", "data": "synthetic (random-init weights N(0, 0.02), random token ids)"}))
    return 0


def bench_calibrate_mfma(args, dev, stream) -> int:
    """K launches of the pure-MFMA calibration kernel (256 workgroups of 4 waves, each wave
    4 x 8192 MFMAs of 32x32x16 bf16) between two events; prints its achieved TFLOP/s."""
    import ctypes

    import torch
    from paper_2602_06161_amd import cover
    from paper_2602_06161_amd.build import LIB_TIMING

    cover.use_library(LIB_TIMING)
    grid, iters = 256, 8192
    out = torch.empty(grid * 256, device=dev, dtype=torch.float32)
    fn = cover.lib().cover_calib_mfma
    fn.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_void_p]
    fn.restype = ctypes.c_int
    run = lambda: fn(cover._ptr(out), grid, iters, cover._stream(stream))
    for _ in range(max(1, args.warmup)):
        if run() != 0:
            raise RuntimeError("calibration launch failed")
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        run()
    e1.record(stream)
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / args.steps
    flops = grid * 4 * 4 * iters * 32768
    print(json.dumps({"calibrate_mfma": "256 workgroups x 4 waves, 4 x 8192 bf16 32x32x16 MFMAs per wave",
                      "flops_per_launch": flops, "us_per_launch": round(us, 3),
                      "tflops": round(flops / us / 1e6, 1),
                      "frac_of_2516_6": round(flops / us / 1e6 / PEAK_BF16_TFLOPS, 4)}))
    return 0


def bench_phase_timing(args, dev, stream) -> int:
    """Per-phase cycle counts of cover_attn_w4_kernel from its timing build: every wave's
    shader-clock stamps at fixed points (see the slot list in the kernel source), summarised
    as medians over all waves of all workgroups, per-step medians, the slowest workgroup, and
    the shader clock (stamps over the 100-MHz real-time counter)."""
    import numpy as np
    import torch
    from paper_2602_06161_amd import cover, synth
    from paper_2602_06161_amd.build import LIB_TIMING

    cover.use_library(LIB_TIMING)
    a = synth.attn_inputs(args.workload, seed=args.seed)
    c = a["cfg"]
    if args.zero_seeds:  # the same launch with empty seed lists (what the seeds cost)
        a["n_seed"] = a["n_seed"] * 0
    t = {k: a[k].to(dev) for k in ("q", "k_live", "v_live", "k_cache", "v_cache", "seed_idx",
                                   "n_seed")}
    attn = cover.PreparedAttn(t["q"], t["k_live"], t["v_live"], t["k_cache"], t["v_cache"],
                              t["seed_idx"], t["n_seed"], stream=stream)
    settle_clocks(attn, args.settle_ms)
    for _ in range(args.warmup):
        attn()
    torch.cuda.synchronize()
    attn()
    torch.cuda.synchronize()
    WG, W, S = 4096, 4, 96
    buf = np.zeros(WG * W * S, dtype=np.uint64)
    rc = cover.lib().cover_attn_timing_read(buf.ctypes.data_as(__import__("ctypes").c_void_p),
                                            __import__("ctypes").c_int64(buf.size))
    if rc != 0:
        raise RuntimeError(f"cover_attn_timing_read failed ({rc})")
    n_qt = -(-c.L // 128)
    nwg = min(WG, c.B * c.Hq * n_qt)
    T = buf.reshape(WG, W, S)[:nwg].astype(np.int64)
    n_it = -(-c.L // 64)
    med = lambda x: float(np.median(x))
    ghz = (T[:, :, 94] - T[:, :, 0]) / ((T[:, :, 95] - T[:, :, 1]) / 100e6) / 1e9
    last_top = 6 + min(n_it - 2, 63)
    phases = {
        "q_k0_landed": T[:, :, 2] - T[:, :, 0],
        "seed_bitmap": T[:, :, 3] - T[:, :, 2],
        "q_to_registers": T[:, :, 4] - T[:, :, 3],
        "s0_and_maxima": T[:, :, 5] - T[:, :, 4],
        "first_step_wait": T[:, :, 6] - T[:, :, 5],
        "steps": T[:, :, last_top] - T[:, :, 6],
        "to_last_stage": T[:, :, 70] - T[:, :, last_top],
        "last_stage": T[:, :, 71] - T[:, :, 70],
        "drain_loads": T[:, :, 72] - T[:, :, 71],
        "merge_exchange": T[:, :, 73] - T[:, :, 72],
        "finish_rows": T[:, :, 74] - T[:, :, 73],
        "issue_stores": T[:, :, 75] - T[:, :, 74],
        "stores_complete": T[:, :, 94] - T[:, :, 75],
        "total": T[:, :, 94] - T[:, :, 0],
    }
    steps = [med(T[:, :, 7 + i] - T[:, :, 6 + i]) for i in range(min(n_it - 2, 63))]
    tot = phases["total"].max(axis=1)
    slow = int(np.argmax(tot))
    # workgroups whose own 128 query rows hold seeds (logical index: query tile li % n_qt of
    # batch row li // (Hq n_qt)) against the others: the launch ends with the slowest
    seeded = np.zeros(nwg, dtype=bool)
    si, ns = a["seed_idx"].numpy(), a["n_seed"].numpy()
    for li in range(nwg):
        b, qt = li // (c.Hq * n_qt), li % n_qt
        pos = si[b, : ns[b]]
        seeded[li] = bool(((pos >= qt * 128) & (pos < qt * 128 + 128)).any())
    split = {}
    for name, sel in (("seeded", seeded), ("other", ~seeded)):
        if sel.any():
            split[name] = {"workgroups": int(sel.sum()),
                           "total_cycles_median": med(tot[sel]),
                           "phase_cycles_median": {k: med(v[sel]) for k, v in phases.items()}}
    rec = {
        "phase_timing": f"{args.workload}: B={c.B} Hq={c.Hq} Hkv={c.Hkv} L={c.L} d={c.d}",
        "workgroups": nwg,
        "sclk_ghz_median": round(med(ghz), 3),
        "sclk_ghz_min": round(float(ghz.min()), 3),
        "cycles_median": {k: med(v) for k, v in phases.items()},
        "cycles_slowest_workgroup": {k: float(v[slow].max()) for k, v in phases.items()},
        "slowest_workgroup": slow,
        "step_cycles_median": steps,
        "seeded_vs_other_workgroups": split,
    }
    print(json.dumps(rec))
    return 0


def bench_block_phase_timing(args, dev, stream) -> int:
    """Per-phase cycle counts of cover_attn_tile_kernel (the single-launch block attention)
    from its timing build, at the LLaDA-8B layer shape: blocks of 256 rows at 768 and 32 rows
    at 992 with the workload's seeds, and 32 rows without seeds.  Medians over all waves of
    all workgroups; per-stage cycles per wave (from its first stage's data to the end of its
    loop, over its own number of stages), for waves 0-3 and 4-7 apart; the merge barrier's
    wait and the workgroup total (first stamp to last)."""
    import ctypes
    import numpy as np
    import torch
    from paper_2602_06161_amd import cover, synth
    from paper_2602_06161_amd.build import LIB_TIMING

    cover.use_library(LIB_TIMING)
    a = synth.attn_inputs("llada", seed=args.seed)
    q, kl, vl, kc, vc, si, ns = (a[k].to(dev) for k in ("q", "k_live", "v_live", "k_cache",
                                                         "v_cache", "seed_idx", "n_seed"))
    B, H, L, d = a["q"].shape
    WG, W, S = 1024, 8, 32
    nst = -(-L // 32)
    cw = [0, 10, 20, 30, 40, 46, 52, 58, 64]  # the kernel's stage split, in 64ths
    n_w = np.array([nst * cw[w + 1] // 64 - nst * cw[w] // 64 for w in range(W)])
    med = lambda x: float(np.median(x))
    for Lq, q_off, seeded in ((256, 768, True), (32, 992, True), (32, 992, False)):
        qb = q[:, :, q_off:q_off + Lq].contiguous()
        call = cover.PreparedRect(qb, kl, vl, kc, vc, q_off, si if seeded else None,
                                  ns if seeded else None, n_split=1, stream=stream)
        settle_clocks(call, args.settle_ms)
        for _ in range(max(1, args.warmup)):
            call()
        torch.cuda.synchronize()
        call()
        torch.cuda.synchronize()
        buf = np.zeros(WG * W * S, dtype=np.uint64)
        rc = cover.lib().cover_rect_timing_read(buf.ctypes.data_as(ctypes.c_void_p),
                                                ctypes.c_int64(buf.size))
        if rc != 0:
            raise RuntimeError(f"cover_rect_timing_read failed ({rc})")
        nwg = min(WG, B * H * -(-Lq // 32))
        T = buf.reshape(WG, W, S)[:nwg].astype(np.int64)
        per_stage = (T[:, :, 20] - T[:, :, 3]) / np.maximum(n_w, 1)[None, :]
        rec = {
            "phase_timing": f"block attention, LLaDA-8B layer B={B} H={H} L={L} d={d}, block of "
                            f"{Lq} rows at {q_off}, {'%d seeds' % int(a['n_seed'][0]) if seeded else 'no seeds'}",
            "workgroups": nwg, "stages_per_wave": n_w.tolist(),
            "cycles_median": {
                "seeds_and_q_landed": med(T[:, :, 1] - T[:, :, 0]),
                "seed_bitmap": med(T[:, :, 2] - T[:, :, 1]),
                "first_stage_landed": med(T[:, :, 3] - T[:, :, 2]),
                "per_stage_waves_0_3": med(per_stage[:, :4]),
                "per_stage_waves_4_7": med(per_stage[:, 4:]),
                "merge_barrier_wait": med(T[:, :, 21] - T[:, :, 20]),
                "merge": med(T[:, :, 22] - T[:, :, 21]),
                "workgroup_total": med(T[:, :, 22].max(axis=1) - T[:, :, 0].min(axis=1)),
            },
            "cycles_max": {
                "first_stage_landed": float((T[:, :, 3] - T[:, :, 2]).max()),
                "merge_barrier_wait": float((T[:, :, 21] - T[:, :, 20]).max()),
            },
        }
        print(json.dumps(rec), flush=True)
    return 0


def bench_block(args, dev, stream) -> int:
    """cover_attn_rect at the LLaDA-8B layer shape (B=1, 32 heads of 128, L=1024): the
    generated block of 256 rows and prefix-cache block sizes of 64 and 32 rows against all
    1024 keys (Sec. 6.6), inputs resident.  Prints one JSON line per block size with the
    launch time (one launch, or the split and merge kernels for n_split > 1; HIP events over
    back-to-back calls) and the roofline of an HBM-bound call: algorithmic bytes = K and V of all keys (seed rows from the cache) + the
    block's q and out + lse."""
    import torch
    from paper_2602_06161_amd import cover, synth

    a = synth.attn_inputs("llada", seed=args.seed)
    q, kl, vl, kc, vc, si, ns = (a[k].to(dev) for k in ("q", "k_live", "v_live", "k_cache",
                                                         "v_cache", "seed_idx", "n_seed"))
    B, H, L, d = a["q"].shape
    K = max(1, args.steps)
    for Lq, q_off in ((256, 768), (64, 896), (32, 992)):
        qb = q[:, :, q_off:q_off + Lq].contiguous()
        # arguments marshalled once: a call is one C-ABI call, so the loop is not bound by
        # Python's per-call overhead (about 12 us, near the kernel's own time)
        call = cover.PreparedRect(qb, kl, vl, kc, vc, q_off, si, ns, stream=stream)
        n = call.n_split
        settle_clocks(call, args.settle_ms)
        for _ in range(max(1, args.warmup)):
            call()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(K):
            call()
        e1.record(stream)
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / K
        alg = B * H * L * d * 2 * 2 + 2 * B * H * Lq * d * 2 + B * H * Lq * 4
        rec = 2 * cover.rect_workspace(B, H, Lq, n) * 4
        flops = 4 * B * H * Lq * L * d
        gbs = alg / us / 1e3
        print(json.dumps({
            "workload": f"block attention, LLaDA-8B layer B={B} H={H} L={L} d={d}, block of {Lq} "
                        f"rows at {q_off}, {int(a['n_seed'][0])} seeds",
            "Lq": Lq, "n_split": n, "steps": K, "us_per_call": round(us, 3),
            "tflops": round(flops / us / 1e6, 1), "split_record_bytes": rec,
            "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": 8000.0, "unit": "GB/s",
                         "frac": round(gbs / 8000.0, 4), "algorithmic_bytes_per_call": alg},
            "dtype": "bf16", "data": "synthetic (seeded N(0,1) q/k/v/cache)"}))
    return 0


def decode_loop(args, dev, stream, model, emb, lm_head, kv, as4, tokens, L, prompt, gen, mask_id,
                max_seeds, cap, n_layers) -> int:
    """COVER decoding of the 256-position block from all-[MASK] to completion on the random
    model (Sec. 3 loop; Sec. 5.1-5.3 each step): the previous step's seeds enter as [MASK] and
    read their K/V from the previous step's buffers, then token statistics, the state update
    (drafting with cap 15 over tau 0.9, Keep/Replace/ReMask), the attention masses and the
    next seeds.  The LM head is scaled by --lm-scale so that confidences spread over (0, 1]
    (random weights otherwise give near-uniform distributions that never pass tau).  Reports
    the step count T, the revision statistics and flip-flops F (Sec. 4), and checks the
    Lemma A.1 bound T >= ceil((L + F) / B) and the unmask-count identity
    sum_t |D_t| = L + #ReMask at completion.

    Semi-autoregressive order (Sec. 6.1): drafting is restricted to the current block of
    --block-len positions (confidences outside it are NaN: never drafted): the first block
    that still holds a [MASK], so a block reopened by a ReMask is finished before the next;
    revision and seed selection cover the whole generated region.  --min-draft
    (default 1) drafts the most confident masked positions of the block when none passes
    tau; 0 is the paper's rule, under which a random model can stall.  --temperature T > 0
    replaces the argmax predictions and their probabilities by temperature samples
    (cover_token_sample, seeded by --seed and the step index), for drafting and revision.

    --variant wo_kv: verification by masking the seeds in the input only (no KV override and
    no diagonal rule: the attention is called without seeds).  --variant wo_seed: the seeds
    are ranked by their confidence drop, log p at drafting minus log p now (same selection
    kernel and budget rule, with zero attention masses)."""
    import numpy as np
    import torch
    from paper_2602_06161_amd import cover

    tau, budget = args.tau, args.remask_budget  # Sec. 6.1: 0.9 and about 5
    prompt_ids = torch.from_numpy(tokens[:prompt]).to(dev)
    tok = torch.full((1, gen), mask_id, dtype=torch.int32, device=dev)
    cnt = torch.zeros((1, gen), dtype=torch.int32, device=dev)
    last = torch.full((1, gen), -1, dtype=torch.int32, device=dev)
    seed_idx = torch.full((1, max_seeds), -1, dtype=torch.int32, device=dev)
    n_seed = torch.zeros(1, dtype=torch.int32, device=dev)
    trash = torch.tensor([L], device=dev)
    no_seeds = torch.zeros(1, dtype=torch.int32, device=dev)
    logp_draft = torch.zeros((1, gen), dtype=torch.float32, device=dev)
    zeros = torch.zeros((1, gen), dtype=torch.float32, device=dev)
    tot = np.zeros(6, np.int64)  # |D|, kept, replaced, remasked, (unused), flip-flops
    blk = max(1, min(args.block_len, gen))
    pos = torch.arange(gen, device=dev)
    cur = 0  # current block
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    T, done, idle = 0, False, 0
    while T < args.max_steps and not done and idle < 32:
        parity = T & 1
        # model input: the prompt and the state, previous seeds fed as [MASK] (Sec. 5.1)
        ids = torch.cat((prompt_ids, tok[0].long(), trash))
        ids[torch.where(seed_idx[0] >= 0, seed_idx[0].long(), trash)] = mask_id
        attn_n = no_seeds if args.variant == "wo_kv" else n_seed
        logits, lse, q_last = model(ids[:L], parity, seed_idx, attn_n, False)
        logits = logits * args.lm_scale
        if args.temperature > 0:  # stochastic decoding: sampled tokens and their probabilities
            am, conf = cover.cover_token_sample(logits, args.temperature, args.seed, T,
                                                stream=stream)
        else:
            _, conf, am = cover.cover_token_stats(logits, want_logp=False, stream=stream)
        in_blk = (pos >= cur * blk) & (pos < (cur + 1) * blk)
        conf_blk = torch.where(in_blk, conf, torch.full_like(conf, float("nan")))  # never drafted
        flags, drafted, counts, ff = cover.cover_decode_update(
            tok, am[None], conf_blk[None], seed_idx, n_seed, cnt, mask_id, tau, cap, budget,
            prompt, last_unmask=last, min_draft=args.min_draft, stream=stream)
        logp, _, _ = cover.cover_token_stats(logits, tok[0], want_conf=False, want_argmax=False,
                                             stream=stream)
        masked = (tok == mask_id).to(torch.uint8)  # M_t, after the update (Sec. 5.3 d_in)
        if args.variant == "wo_seed":
            # confidence drop since drafting: log p at the unmasking minus log p now
            logp_draft = torch.where(drafted == 1, logp[None], logp_draft)
            cover.cover_select_seeds(logp[None] - logp_draft, zeros, zeros, flags, max_seeds,
                                     prompt, seed_idx=seed_idx, n_seed=n_seed, want_score=False,
                                     stream=stream)
        else:
            k_cur, _ = kv[parity][n_layers - 1]
            k_prev, _ = kv[1 - parity][n_layers - 1]
            d_in, d_out = cover.cover_attn_stats(as4(q_last), as4(k_cur), as4(k_prev), seed_idx,
                                                 attn_n, lse, masked, drafted, prompt,
                                                 stream=stream)
            cover.cover_select_seeds(logp[None], d_in, d_out, flags, max_seeds, prompt,
                                     seed_idx=seed_idx, n_seed=n_seed, want_score=False,
                                     stream=stream)
        c = counts[0].cpu().numpy()
        tot[:4] += c[:4]
        tot[5] += int(ff[0].item())
        T += 1
        done = c[4] == 0
        if not done:  # the first block that still holds a [MASK] (a ReMask can reopen one)
            cur = int(torch.argmax((tok[0] == mask_id).to(torch.int32)).item()) // blk
        idle = idle + 1 if c[0] == 0 and c[3] == 0 else 0  # no draft and no ReMask: no progress
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    F = int(tot[5])
    revisions = int(tot[2] + tot[3])
    bound = -(-(gen + F) // cap)
    print(json.dumps({
        "workload": f"{args.variant} decoding loop, random-init LLaDA-8B-shaped model (32 "
                    f"layers), B=1, prompt {prompt} + block {gen} from all [MASK], tau {tau}, cap {cap}, "
                    f"ReMask budget {budget}, {max_seeds} seeds max, blocks of {blk}, "
                    f"min_draft {args.min_draft}, temperature {args.temperature}, "
                    f"LM head x{args.lm_scale}",
        "steps": T, "terminated": bool(done), "stalled": idle >= 32, "wall_s": round(wall, 3),
        "ms_per_step": round(wall * 1e3 / T, 3), "tokens_per_s": round(gen / wall, 1),
        "drafted": int(tot[0]), "kept": int(tot[1]), "replaced": int(tot[2]),
        "remasked": int(tot[3]), "flip_flops": F, "total_revisions": revisions,
        "effective_revisions": int(tot[2] + tot[3] - F),
        "effective_revision_ratio": round((tot[2] + tot[3] - F) / revisions, 4) if revisions else None,
        "lemma_a1_bound": bound, "lemma_a1_holds": bool(T >= bound) if done else None,
        "unmask_identity_holds": bool(tot[0] == gen + tot[3]) if done else None,
        "dtype": "bf16", "data": "synthetic (random-init weights, random prompt ids)"}))
    return 0


def cpu_baseline(a: dict, flops: int) -> dict:
    """The fp64 oracle (as is) on the same step: full attention layer (fast mode) plus the
    selection, repeated until ~10 s have elapsed (at most 200 repetitions)."""
    import numpy as np
    import oracle

    args = [oracle._f64(a[k]) for k in ("q", "k_live", "v_live", "k_cache", "v_cache")]
    si, ns = a["seed_idx"].numpy(), a["n_seed"].numpy()
    sel = [a[k].numpy() for k in ("logp", "d_in", "d_out", "flags")]
    reps, t_total = 0, 0.0
    while (t_total < 10.0 and reps < 200) or reps == 0:
        t0 = time.perf_counter()
        oracle.attn(*args, si, ns, scale=a["scale"], mode="fast")
        oracle.select(*sel, a["cfg"].n_seeds, a["pos_offset"])
        t_total += time.perf_counter() - t0
        reps += 1
    per = t_total / reps
    cores = oracle.threads()
    # one core: the attention of one head (all L rows), about 2 s of repetitions
    c = a["cfg"]
    rows = np.arange(c.L, dtype=np.int64)
    oracle.set_threads(1)
    try:
        reps1, t1 = 0, 0.0
        while (t1 < 2.0 and reps1 < 100) or reps1 == 0:
            t0 = time.perf_counter()
            oracle.attn(*args, si, ns, scale=a["scale"], mode="fast", rows=rows)
            t1 += time.perf_counter() - t0
            reps1 += 1
    finally:
        oracle.set_threads(cores)
    flops1 = 4 * c.L * c.L * c.d
    return {"value": round(flops / per / 1e12, 5), "unit": "TFLOP/s", "cores": cores,
            "kind": "oracle", "seconds_per_step": round(per, 4),
            "sample": f"{reps} full layer-steps (all {c.Hq} heads x {c.L} rows, fp64, "
                      f"fast mode) + selection, {t_total:.1f} s total",
            "single_core": {"value": round(flops1 * reps1 / t1 / 1e12, 6), "unit": "TFLOP/s",
                            "cores": 1, "sample": f"{reps1} x the attention of one head "
                                                  f"({c.L} rows x {c.L} keys, fp64, fast mode), "
                                                  f"{t1:.1f} s"}}


if __name__ == "__main__":
    sys.exit(main())
