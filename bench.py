#!/usr/bin/env python3
"""Decode-step benchmark: one persistent-kernel decode step on one MI355X.

Default workload: a Llama-2-7B-shaped decoder (32 layers, hidden 4096, 32 heads of 128 (MHA),
SwiGLU 11008, vocab 32000, untied LM head), random bf16 weights N(0, 0.02), batch 1, KV
prefilled to context 1024, greedy decode: the largest batch-1 workload. A "step" generates one
token per lane: embedding, all layers, final norm, LM head and argmax, in one kernel launch.
Step t feeds its greedy token to step t+1 on the device; positions and cache lengths (S + t)
are uploaded before the timed region.

Printed as one JSON line: latency per step (us/token), Eq. 2 bytes and MBU against the
8 TB/s HBM3E peak, a roofline object for the kernel, the per-stage multi-launch ablation on the
same inputs, the CPU reference decoder timed on a bounded sample on this host, and the same
latency and MBU for the other batch-1 cells of the 7B-13B class (Qwen3-8B and Llama-2-13B
shapes at context 2048), measured in the same run.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "decode step latency (µs/token) and MBU % of MI355X HBM peak, batch 1"
PEAK_GBS = 8000.0


def kernel_source_hash() -> str:
    import glob
    import hashlib
    h = hashlib.sha256()
    for f in sorted(glob.glob(os.path.join(ROOT, "paper_2609_12379_amd", "csrc", "*"))):
        if f.endswith((".h", ".hip", ".cpp")):
            with open(f, "rb") as fh:
                h.update(fh.read())
    return h.hexdigest()[:16]


def profiled_traffic(config_name: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary of this workload, if
    it was taken on the current kernel sources (else None)."""
    path = os.path.join(ROOT, "profiles", f"step_kernel_{config_name}.md")
    if not os.path.exists(path):
        return None
    fields = {}
    with open(path) as f:
        for line in f:
            line = line.strip()
            if ":" in line and line.split(":", 1)[0] in ("source_hash", "traffic_bytes_per_launch",
                                                          "fetch_bytes_per_launch", "write_bytes_per_launch"):
                k, v = line.split(":", 1)
                fields[k] = v.strip()
    if fields.get("source_hash") != kernel_source_hash():
        return None
    return {k: int(v) for k, v in fields.items() if k != "source_hash"}


def measure(name: str, args, context: int = 0, cpu: bool = False, ablation: bool = False) -> dict:
    """Times one workload and releases every device buffer it allocated before returning."""
    import gc
    import torch
    from synthetic import get_config, make_workload, as_u16
    from paper_2609_12379_amd.fm import Decoder, plan_query
    from paper_2609_12379_amd.metrics import step_bytes

    cfg0 = get_config(name)
    if context:
        cfg0 = dict(cfg0, ctx=(context, context))
    total_steps = args.warmup + args.steps
    t_gen = time.time()
    # weights and KV prefill are drawn on the device (seeded, same distributions as the host recipe)
    wl = make_workload(cfg0, steps=max(total_steps, cfg0["steps"]), device="cuda")
    cfg = wl.cfg
    gen_s = time.time() - t_gen
    b = cfg["batch"]

    wdev = {k: v for k, v in wl.weights.items() if k != "layers" and v is not None}
    wdev["layers"] = list(wl.weights["layers"])
    kc, vc = list(wl.kcache), list(wl.vcache)
    dec = Decoder(cfg, wdev, kc, vc, n_workgroups=args.nwg, attn_items=args.attn_items, dyn_chunk_kb=args.dyn_chunk_kb)

    S = wl.S
    pos_all = torch.tensor([[s + t for s in S] for t in range(total_steps)], dtype=torch.int32, device="cuda")
    logits = torch.empty((b, cfg["vocab"]), dtype=torch.float32, device="cuda")
    ids = torch.empty((total_steps + 1, b), dtype=torch.int32, device="cuda")
    ids[0] = torch.tensor(wl.start, dtype=torch.int32)

    def run(t, multilaunch=False):
        dec.step(ids[t], pos_all[t], pos_all[t], logits, ids[t + 1], multilaunch=multilaunch)

    for t in range(args.warmup):
        run(t)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    w0 = time.perf_counter()
    e0.record(stream)
    for t in range(args.warmup, total_steps):
        run(t)
    e1.record(stream)
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - w0) * 1e3
    ev_ms = e0.elapsed_time(e1)
    ms_per_step = ev_ms / args.steps
    assert dec.last_error() == 0, "device reported an error"
    assert bool(torch.isfinite(logits).all()), "non-finite logits"

    # Eq. 2 bytes of each timed step: attention reads kv_len + 1 slots per lane.
    bytes_steps = [step_bytes(cfg, [s + t + 1 for s in S]) for t in range(args.warmup, total_steps)]
    mean_bytes = sum(bytes_steps) / len(bytes_steps)
    achieved_gbs = mean_bytes / (ms_per_step * 1e-3) / 1e9
    mbu = sum(bytes_steps) / (ev_ms * 1e-3) / (PEAK_GBS * 1e9)

    # Two-point slope (the paper's latency estimate): min over replicates of
    # (t(N2) - t(N1)) / (N2 - N1), steps replayed from the warm state.
    def timed(n, multilaunch=False):
        torch.cuda.synchronize()
        a, c = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for t in range(n):
            run(args.warmup + t, multilaunch)
        c.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(c)

    n2 = args.steps
    n1 = max(1, n2 // 4)
    slope_ms = min((timed(n2) - timed(n1)) / (n2 - n1) for _ in range(3))

    ctx = S if len(set(S)) > 1 else S[0]
    res = {
        "workload": f"{cfg['name']}-shaped decoder, b{b}, context {ctx}, greedy decode",
        "cfg": cfg, "S": S,
        "ms_per_step": ms_per_step, "ev_ms": ev_ms, "wall_ms": wall_ms,
        "mean_bytes": mean_bytes, "achieved_gbs": achieved_gbs, "mbu": mbu, "slope_ms": slope_ms,
        "setup_s": gen_s, "bytes_steps": bytes_steps,
    }

    if ablation:
        # Per-stage multi-launch ablation: the same step kernel launched once per operator
        # stage (per layer QKV, attention, O projection, gate/up, down; then the LM head).
        for t in range(2):
            run(args.warmup + t, True)
        torch.cuda.synchronize()
        ml = timed(args.steps, True) / args.steps
        res["ablation"] = {
            "baseline": "per-stage multi-launch: the step kernel launched once per operator stage "
                        "(QKV, attention, O projection, gate/up, down per layer, then the LM head); each "
                        "launch keeps the fusions inside its stage (norm, QK-norm, RoPE, KV append, merge)",
            "ms_per_step": round(ml, 5), "us_per_token": round(ml * 1e3, 2),
            "mbu_pct": round(100 * sum(bytes_steps) / (ml * args.steps * 1e-3) / (PEAK_GBS * 1e9), 2),
            "launches_per_step": plan_query(cfg, 256).n_stages,
            "megakernel_speedup": round(ml / ms_per_step, 3)}

    if cpu:
        # CPU reference decoder on this host: a bounded sample of the same workload.
        from oracle.oracle import Oracle
        wu = {k: as_u16(v.cpu()) for k, v in wl.weights.items() if k != "layers" and v is not None}
        wu["layers"] = [{k: as_u16(v.cpu()) for k, v in lw.items()} for lw in wl.weights["layers"]]
        orc = Oracle(cfg, wu)
        # the device arenas were advanced by the timed steps; the oracle starts from the prefill,
        # which is untouched below each lane's context S_i
        kco = [as_u16(t.cpu()).copy() for t in wl.kcache]
        vco = [as_u16(t.cpu()).copy() for t in wl.vcache]
        threads = int(os.environ.get("OMP_NUM_THREADS", len(os.sched_getaffinity(0))))
        tok = list(wl.start)
        n_cpu, t_cpu, span = 0, 0.0, cfg["max_ctx"] - max(S)
        while n_cpu < 2 or t_cpu < args.cpu_seconds:
            t = n_cpu % span            # replay from the start once the cache bound is reached
            if t == 0:
                tok = list(wl.start)
            pos = [s + t for s in S]
            c0 = time.perf_counter()
            r = orc.step(kco, vco, tok, pos, pos, precision="f32")
            t_cpu += time.perf_counter() - c0
            tok = [int(v) for v in r.next_ids]
            n_cpu += 1
        model = ""
        try:
            with open("/proc/cpuinfo") as f:
                for line in f:
                    if line.startswith("model name"):
                        model = line.split(":", 1)[1].strip()
                        break
        except OSError:
            pass
        res["cpu_baseline"] = {"value": round(t_cpu / n_cpu * 1e6, 1), "unit": "us/token", "cores": threads,
                               "kind": "oracle", "cpu_model": model,
                               "sample": f"{n_cpu} greedy steps of the same workload, replayed from the start "
                                         f"every {span} steps (fp32 oracle, {t_cpu:.1f} s of CPU time)"}
        del orc, wu, kco, vco

    # Release the handle and every device tensor before the next workload (or the process's
    # exit): nothing of this workload is left to interpreter teardown.
    dec.close()
    del dec, wdev, kc, vc, wl, pos_all, logits, ids
    gc.collect()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=64)
    ap.add_argument("--warmup", type=int, default=64)
    ap.add_argument("--config", default="llama2-7b")
    ap.add_argument("--extra", default="qwen3-8b-b1,llama2-13b-b1",
                    help="other workloads timed in the same run (comma-separated; empty for none)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU reference leg")
    ap.add_argument("--no-ablation", action="store_true", help="skip the multi-launch ablation")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="budget of the CPU sample")
    ap.add_argument("--calib-copy-mb", type=int, default=0,
                    help="also run a plain device copy of this many MiB (counter calibration)")
    ap.add_argument("--nwg", type=int, default=0)
    ap.add_argument("--attn-items", type=int, default=0)
    ap.add_argument("--dyn-chunk-kb", type=int, default=0,
                    help="weight KiB per dynamically claimed GEMV chunk (0 automatic, -1 fixed tiles only)")
    ap.add_argument("--context", type=int, default=0,
                    help="prefilled context of every lane, overriding the workload's (a context sweep)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)

    import torch
    from paper_2609_12379_amd.fm import load

    load()  # fail loudly if the HIP library is missing
    assert torch.cuda.is_available(), "bench.py needs the GPU"

    m = measure(args.config, args, context=args.context, cpu=not args.no_cpu, ablation=not args.no_ablation)
    cfg, S = m["cfg"], m["S"]
    b = cfg["batch"]
    out = {
        "metric": METRIC,
        "value": round(m["ms_per_step"] * 1e3, 2),
        "unit": "us/token",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(m["ms_per_step"], 5),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "storage": "bf16 weights and KV cache",
        "data": "synthetic",
        "config": {"workload": m["workload"],
                   "layers": cfg["n_layers"], "hidden": cfg["hidden"], "heads": [cfg["n_heads"], cfg["n_kv_heads"]],
                   "head_dim": cfg["head_dim"], "intermediate": cfg["intermediate"], "vocab": cfg["vocab"],
                   "batch": b, "context": S, "timing_scope": "step with greedy argmax, inputs resident in HBM"},
        "mbu_pct": round(100 * m["mbu"], 2),
        "bytes_per_step_eq2": int(m["mean_bytes"]),
        "two_point_slope_us": round(m["slope_ms"] * 1e3, 2),
        "wall_ms_timed_region": round(m["wall_ms"], 3),
        "roofline": {"bound": "hbm", "achieved": round(m["achieved_gbs"], 1), "peak": PEAK_GBS, "unit": "GB/s",
                     "frac": round(m["achieved_gbs"] / PEAK_GBS, 4), "traffic": None,
                     "kernel": "fm::dev::step_kernel (one launch per step)"},
    }
    tr = None if args.context else profiled_traffic(cfg["name"])
    if tr is not None:
        out["roofline"]["traffic"] = tr["traffic_bytes_per_launch"]
        out["read_amplification_rho"] = round(tr["fetch_bytes_per_launch"] / m["mean_bytes"], 4)
    if "ablation" in m:
        out["ablation_per_stage_multilaunch"] = m["ablation"]
    if "cpu_baseline" in m:
        out["cpu_baseline"] = m["cpu_baseline"]
    out["setup_s"] = round(m["setup_s"], 1)

    if args.calib_copy_mb:
        n = args.calib_copy_mb * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        out["calib_copy_bytes_each_way"] = n * 4
        del src, dst

    extras = [e for e in args.extra.split(",") if e and e != args.config] if not args.context else []
    if extras:
        cells = {}
        for e in extras:
            r = measure(e, args)
            cells[e] = {"workload": r["workload"], "us_per_token": round(r["ms_per_step"] * 1e3, 2),
                        "mbu_pct": round(100 * r["mbu"], 2), "bytes_per_step_eq2": int(r["mean_bytes"]),
                        "two_point_slope_us": round(r["slope_ms"] * 1e3, 2)}
        out["other_batch1_cells"] = cells
    print(json.dumps(out), flush=True)
    torch.cuda.synchronize()


if __name__ == "__main__":
    main()
