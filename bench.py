"""Benchmark of the sharded expert-FFN MoE layer on one MI355X.

One step = one full layer forward (route -> dispatch -> expert FFN shard -> combine, as
MoEShardLayer.forward issues it) over one batch of synthetic tokens already resident in
HBM, every timed step after a 512 MiB write + read-back cache flush.  Prints one JSON line.

  python bench.py [--steps K] [--warmup W] [--config c5] [--no-cpu-baseline] [--warm-steps N]
  python bench.py --ablation        # grouped vs per-expert launches, E = 8 .. 256

HBM traffic of the expert-FFN kernels comes from two rocprofv3 counter runs of this script,
one with --pmc FETCH_SIZE and one with --pmc WRITE_SIZE, each with --copy-probe-mib so that
the same run also holds a plain copy of known size (an elementwise negation, read N bytes,
write N bytes) that calibrates the counter:

  rocprofv3 --pmc FETCH_SIZE --output-format csv -d DIR_F -o run -- python3 bench.py \
      --no-cpu-baseline --steps 3 --warmup 1 --copy-probe-mib 256
  (the same with WRITE_SIZE into DIR_W)
  python bench.py --config c2 --summarize-counters DIR_F DIR_W   # -> profiles/ffn_traffic_c2.json

MFMA work and busy fraction of the same kernels come from one more counter run:

  rocprofv3 --pmc SQ_INSTS_VALU_MFMA_MOPS_BF16 SQ_INSTS_VALU_MFMA_MOPS_F32 SQ_VALU_MFMA_BUSY_CYCLES \
      GRBM_GUI_ACTIVE --output-format csv -d DIR -o run -- python3 bench.py --config c4 \
      --no-cpu-baseline --steps 3 --warmup 1
  python bench.py --config c4 --summarize-mfma DIR                # -> profiles/mfma_c4.json
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import synth  # noqa: E402

PEAK_HBM_GBS = 8000.0
PEAK_BF16_TFLOPS = 2500.0
PEAK_F32_TFLOPS = 157.3
FFN_SOURCES = ["paper_2503_08467_amd/csrc/ffn.hip", "paper_2503_08467_amd/csrc/common.h",
               "paper_2503_08467_amd/csrc/lds_dma.h", "paper_2503_08467_amd/csrc/kernels.h"]


def ffn_source_hash() -> str:
    """Hash of the expert-step sources as the compiler sees them: line comments and blank
    lines left out, so that a comment edit does not orphan the committed counter figures."""
    h = hashlib.sha256()
    for p in FFN_SOURCES:
        with open(os.path.join(ROOT, p), encoding="utf-8") as fh:
            for line in fh:
                code = line.split("//", 1)[0].rstrip()
                if code:
                    h.update(code.encode() + b"\n")
    return h.hexdigest()[:16]


def measured_traffic(config: str):
    """HBM bytes per FFN call from the committed rocprofv3 counter summary, if it was taken
    on the current FFN source; else None."""
    path = os.path.join(ROOT, "profiles", f"ffn_traffic_{config}.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        rec = json.load(fh)
    if rec.get("ffn_source_hash") != ffn_source_hash():
        return None
    return rec.get("hbm_bytes_per_call")


def is_ffn_kernel(name: str) -> bool:
    """The kernels of the expert step: the grouped GEMMs (up- and down-projection) and, for
    small bf16 calls whose down-projection splits K, the sum of its parts."""
    return any(k in name for k in ("gemm_bf16", "gemm_up_pairs", "gemm_f32", "split_reduce"))


def is_layer_kernel(name: str) -> bool:
    """Kernels of a layer step (route, dispatch, expert step, combine), not weight packing,
    uploads or the copy probe."""
    return is_ffn_kernel(name) or any(k in name for k in ("route", "dispatch_", "combine_kernel"))


def stage_bytes(cfg, fused_gather: bool, top1_fused: bool, bias_per_row: bool) -> dict:
    """Algorithmic HBM bytes of route, dispatch and combine for one layer call: each input
    read once and each output written once."""
    T, k, E, h, A = cfg.T, cfg.k, cfg.E, cfg.h, cfg.A
    es = 2 if cfg.dtype == "bf16" else 4
    route = T * h * es + E * h * es + (T * E * 4 if bias_per_row else E * 4) + T * k * 8
    dispatch = 3 * A * 4 + (2 * E + 1) * 4 + (0 if fused_gather else 2 * A * h * es)
    combine = 0 if top1_fused else A * h * es + T * h * es + T * k * 8
    return {"route": route, "dispatch": dispatch, "combine": combine}


def ffn_matrix(name: str) -> str:
    """"down" for the down-projection launches (epilogue template argument 3, no activation;
    the sum of its K parts), else "up"."""
    if "split_reduce" in name:
        return "down"
    return "down" if re.search(r"<(?:[^>]*, )?3, (?:true|false)(?:, \d+)?>", name) else "up"


def summarize_counters(config: str, fetch_dir: str, write_dir: str, probe_mib: int):
    """Per-call HBM bytes of the expert-FFN launches from two rocprofv3 counter runs.

    Each counter (KiB per dispatch) is scaled by known_bytes / counter for the copy probe of
    the same run.  One FFN call is one launch of each grouped-GEMM instantiation that appears
    (up-projection with activation, down-projection)."""
    import csv
    import glob
    known = probe_mib * 1024 * 1024

    def read(d, counter):
        per = {}
        for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            for r in csv.DictReader(open(f)):
                if r["Counter_Name"] != counter:
                    continue
                per.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]) * 1024.0)
        probe = [v for k, vs in per.items() if "neg" in k for v in vs]
        gemm = {k: float(np.mean(v)) for k, v in per.items() if is_ffn_kernel(k)}
        other = {k: float(np.mean(v)) for k, v in per.items() if is_layer_kernel(k) and not is_ffn_kernel(k)}
        if not probe or not gemm:
            raise SystemExit(f"{d}: missing copy probe or expert-FFN launches for {counter}")
        factor = known / float(np.median(probe))
        return factor, {k: v * factor for k, v in gemm.items()}, {k: v * factor for k, v in other.items()}

    ff, fetch, fetch_o = read(fetch_dir, "FETCH_SIZE")
    wf, write, write_o = read(write_dir, "WRITE_SIZE")
    cmd = ("rocprofv3 --pmc {c} --output-format csv -d {d} -o run -- python3 bench.py --config " + config +
           " --no-cpu-baseline --steps 3 --warmup 1 --copy-probe-mib " + str(probe_mib))
    rec = {"config": config, "ffn_source_hash": ffn_source_hash(),
           "commands": [cmd.format(c="FETCH_SIZE", d=fetch_dir), cmd.format(c="WRITE_SIZE", d=write_dir),
                        f"python bench.py --config {config} --summarize-counters {fetch_dir} {write_dir} "
                        f"--copy-probe-mib {probe_mib}"],
           "note": "FETCH_SIZE and WRITE_SIZE in KiB per dispatch, scaled by the factor that maps the copy "
                   "probe's counter to its known size; one FFN call = both launches",
           "fetch_factor": round(ff, 4), "write_factor": round(wf, 4),
           "fetch_bytes_per_launch": {k: round(v) for k, v in fetch.items()},
           "write_bytes_per_launch": {k: round(v) for k, v in write.items()},
           "hbm_bytes_per_call": round(sum(fetch.values()) + sum(write.values())),
           "other_steps_fetch_bytes_per_launch": {k: round(v) for k, v in fetch_o.items()},
           "other_steps_write_bytes_per_launch": {k: round(v) for k, v in write_o.items()}}
    path = os.path.join(ROOT, "profiles", f"ffn_traffic_{config}.json")
    with open(path, "w") as fh:
        json.dump(rec, fh, indent=1)
    print(json.dumps(rec, indent=1))


MFMA_COUNTERS = ("SQ_INSTS_VALU_MFMA_MOPS_BF16", "SQ_INSTS_VALU_MFMA_MOPS_F32", "SQ_VALU_MFMA_BUSY_CYCLES",
                 "GRBM_GUI_ACTIVE")


def summarize_mfma(config: str, pmc_dir: str, simds: int = 1024, xcds: int = 8):
    """MFMA work and busy fraction of the expert-FFN launches from one rocprofv3 counter run
    (--pmc with MFMA_COUNTERS), beside the algorithmic flops of the same launches.

    Counter flops = MFMA ops x 512.  Busy = SQ_VALU_MFMA_BUSY_CYCLES summed over the SIMDs /
    (GRBM_GUI_ACTIVE of one XCD x SIMDs); GRBM_GUI_ACTIVE comes summed over the XCDs."""
    import csv
    import glob
    per = {}
    for f in glob.glob(os.path.join(pmc_dir, "**", "*counter_collection.csv"), recursive=True):
        for r in csv.DictReader(open(f)):
            k = r["Kernel_Name"]
            if not is_ffn_kernel(k):
                continue
            per.setdefault(k, {}).setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
    if not per:
        raise SystemExit(f"{pmc_dir}: no expert-FFN launches")
    cfg = synth.CONFIGS[config]
    n_up = 2 if cfg.act == "swiglu" else 1
    alg = {"up": 2.0 * n_up * cfg.A * cfg.h * cfg.f, "down": 2.0 * cfg.A * cfg.h * cfg.f}
    out = {}
    for k, cs in per.items():
        m = {c: float(np.mean(v)) for c, v in cs.items()}
        flops = (m.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0.0) + m.get("SQ_INSTS_VALU_MFMA_MOPS_F32", 0.0)) * 512
        which = ffn_matrix(k)
        busy = m["SQ_VALU_MFMA_BUSY_CYCLES"] / (m["GRBM_GUI_ACTIVE"] / xcds * simds)
        out[k] = {"matrix": which, "counter_flops": round(flops), "algorithmic_flops": round(alg[which]),
                  "counter_over_algorithmic": round(flops / alg[which], 4), "mfma_busy": round(busy, 4)}
    cmd = (f"rocprofv3 --pmc {' '.join(MFMA_COUNTERS)} --output-format csv -d {pmc_dir} -o run -- python3 bench.py "
           f"--config {config} --no-cpu-baseline --steps 3 --warmup 1")
    rec = {"config": config, "ffn_source_hash": ffn_source_hash(),
           "commands": [cmd, f"python bench.py --config {config} --summarize-mfma {pmc_dir}"],
           "note": "per launch, averaged over the run's launches; counter flops include the MFMAs of padded rows "
                   "in 32-row blocks that hold a valid row; busy is the MFMA pipes' busy fraction over the "
                   "launch, against the clock the kernel ran at",
           "launches": out}
    path = os.path.join(ROOT, "profiles", f"mfma_{config}.json")
    with open(path, "w") as fh:
        json.dump(rec, fh, indent=1)
    print(json.dumps(rec, indent=1))


def ablation_per_expert(seed: int, reps: int, experts):
    """The grouped single launch against one launch pair per expert (the expert step with
    and without the grouped formulation), on the paper's evaluation shape: b = 250, s = 120
    (30 000 tokens), h = 768, one device's 1/4 shard of a 3072-wide FFN, top-1, skewed
    router with k_r = ceil(0.1 E) hot experts and alpha_r = 0.6.  One JSON line per E."""
    import math
    import torch
    import paper_2503_08467_amd as moe
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream(dev)
    base = synth.CONFIGS["paper128"]
    for E in experts:
        cfg = base.with_(name=f"paper{E}", E=E, routing=("paper", math.ceil(0.1 * E), 0.6))
        L = synth.make(cfg, seed=seed)
        to = lambda a, d=torch.bfloat16: torch.from_numpy(np.ascontiguousarray(a)).to(dev).to(d)
        x, wg, bias = to(L.x), to(L.wg), to(L.sel_bias, torch.float32)
        packed = moe.pack_weights(to(L.w1), to(L.w2), act=cfg.act)
        del L
        idx, w = moe.route(x, wg, cfg.k, bias, False)
        disp = moe.dispatch(idx, x, E)
        out = torch.empty_like(disp.x_perm)
        ws = torch.empty(moe.ffn_workspace_size(cfg.A, packed), dtype=torch.uint8, device=dev)
        touched = int((disp.counts > 0).sum().item())

        def timed(fn):
            for _ in range(3):
                fn()
            torch.cuda.synchronize()
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
            t0 = time.perf_counter()
            ev[0].record(stream)
            for _ in range(reps):
                fn()
            ev[1].record(stream)
            torch.cuda.synchronize()
            return ev[0].elapsed_time(ev[1]) * 1e3 / reps, (time.perf_counter() - t0) * 1e6 / reps

        g_us, g_wall = timed(lambda: moe.expert_ffn_shard(disp.x_perm, disp.offsets, packed, out=out, ws=ws))
        # the per-expert loop reads the counts back on every call, as it must to size its launches
        p_us, p_wall = timed(lambda: moe.expert_ffn_shard_per_expert(disp.x_perm, disp.offsets, packed, out=out,
                                                                     ws=ws))
        print(json.dumps({"ablation": "grouped vs per-expert launches", "experts": E, "tokens": cfg.T,
                          "hidden": cfg.h, "shard_inner_width": cfg.f, "hot_experts": math.ceil(0.1 * E),
                          "touched_experts": touched, "grouped_ffn_us": round(g_us, 1),
                          "per_expert_ffn_us": round(p_us, 1), "per_expert_wall_us": round(p_wall, 1),
                          "speedup": round(p_us / g_us, 2), "launches_grouped": 2,
                          "launches_per_expert": 2 * touched}), flush=True)
        del packed, x, wg, bias, idx, w, disp, out, ws
        torch.cuda.empty_cache()


def cpu_baseline(cfg_name: str, seed: int, budget_s: float = 40.0):
    """The fp64 oracle on a bounded sample of the same workload (its first tokens): the
    sample grows until one run takes a quarter of budget_s, then repeats until the total
    reaches it (about 10-20 s of CPU work)."""
    import oracle
    cfg = synth.CONFIGS[cfg_name]
    L = synth.make(cfg_name, seed=seed)

    def run(n):
        x = L.x[:n]
        bias = None if L.sel_bias is None else L.sel_bias[:n]
        t0 = time.perf_counter()
        idx, w, _ = oracle.route(x, L.wg, cfg.k, bias, cfg.renorm)
        _, offsets, row_src, pos_of = oracle.dispatch(idx, cfg.E)
        y_perm = oracle.expert_ffn(x[row_src], offsets, L.w1, L.w3, L.w2, cfg.act)
        oracle.combine(y_perm, pos_of, w)
        return time.perf_counter() - t0

    n = min(cfg.T, 64)
    dt = run(n)
    while dt < budget_s / 4 and n < cfg.T:
        n = min(cfg.T, max(2 * n, int(n * (budget_s / 2) / max(dt, 1e-3))))
        dt = run(n)
    reps = 1
    while dt < budget_s / 4 and reps < 8:  # whole workload fits: repeat it for a steadier rate
        dt += run(n)
        reps += 1
    return {"value": n * reps / dt, "unit": "tokens/s", "cores": oracle.num_threads(), "cpu": host_cpu_model(),
            "kind": "oracle",
            "sample": f"first {n} of {cfg.T} tokens of workload {cfg_name} x{reps}, full layer "
                      f"(route, dispatch, expert FFN, combine) in fp64, {dt:.1f} s"}


def host_cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", default="c5")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--warm-steps", type=int, default=50,
                    help="after the timed (cold-cache) steps, this many back-to-back steps with warm caches")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="run an untimed plain copy of this size first (counter calibration)")
    ap.add_argument("--summarize-counters", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"))
    ap.add_argument("--summarize-mfma", metavar="PMC_DIR")
    ap.add_argument("--unfused-gather", action="store_true",
                    help="write x_perm in the dispatch step instead of gathering rows in the expert step")
    ap.add_argument("--ablation", action="store_true",
                    help="grouped launch vs one launch pair per expert over E = 8 .. 256 (paper's shape)")
    args = ap.parse_args()
    if args.summarize_counters:
        summarize_counters(args.config, *args.summarize_counters, probe_mib=args.copy_probe_mib or 256)
        return
    if args.summarize_mfma:
        summarize_mfma(args.config, args.summarize_mfma)
        return
    if args.ablation:
        ablation_per_expert(args.seed, reps=max(args.steps // 5, 5), experts=(8, 16, 32, 64, 128, 256))
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: this layer's multi-GPU exchange is not built, so only "
              "--gpus 1 is supported", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2503_08467_amd as moe

    cfg = synth.CONFIGS[args.config]
    L = synth.make(cfg, seed=args.seed)
    dt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    to = lambda a, d=dt: None if a is None else torch.from_numpy(np.ascontiguousarray(a)).to(dev).to(d)
    x, wg = to(L.x), to(L.wg)
    bias = to(L.sel_bias, torch.float32)
    packed = moe.pack_weights(to(L.w1), to(L.w2), to(L.w3), act=cfg.act)
    layer = moe.MoEShardLayer(wg, packed, cfg.k, bool(cfg.renorm), max_tokens=cfg.T,
                              fused_gather=not args.unfused_gather)
    del L.w1, L.w2, L.w3

    stream = torch.cuda.current_stream(dev)
    if args.copy_probe_mib:
        src = torch.ones(args.copy_probe_mib * 1024 * 1024 // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):  # each launch reads probe_mib MiB and writes probe_mib MiB
            torch.neg(src, out=dst)
        torch.cuda.synchronize()
        del src, dst

    top1_fused = cfg.k == 1 and not args.unfused_gather

    def step_parts(ev=None, ffn_ev=None):
        """One layer forward as separate calls, for the measurements that need events between
        them.  ev: 5 events around route, dispatch, expert step and combine (stage breakdown);
        ffn_ev: 2 events around the expert-step call only (the expert step alone: the combine
        stays a call of its own)."""
        T, k = cfg.T, cfg.k
        if ev is None and layer.disp.x_perm is None:
            moe.route_dispatch(x, wg, k, bias, bool(cfg.renorm), out=(layer.idx, layer.w), disp=layer.disp,
                               ws=layer.dws)
        else:
            if ev: ev[0].record(stream)
            moe.route(x, wg, k, bias, bool(cfg.renorm), out=(layer.idx, layer.w))
            if ev: ev[1].record(stream)
            moe.dispatch(layer.idx, x, cfg.E, out=layer.disp, ws=layer.dws)
            if ev: ev[2].record(stream)
        if ffn_ev: ffn_ev[0].record(stream)
        if top1_fused:  # gather, expert step and the top-1 combine in one call
            moe.expert_ffn_shard_top1(x, layer.disp.row_src, layer.w.view(-1), layer.disp.offsets, packed,
                                      out=layer.y, ws=layer.fws)
        elif layer.disp.x_perm is None:  # the expert step gathers the rows (no x_perm round trip)
            moe.expert_ffn_shard_gather(x, layer.disp.row_src, layer.disp.offsets, packed, A_max=T * k,
                                        out=layer.y_perm, ws=layer.fws)
        else:
            moe.expert_ffn_shard(layer.disp.x_perm, layer.disp.offsets, packed, A_max=T * k, out=layer.y_perm,
                                 ws=layer.fws)
        if ffn_ev: ffn_ev[1].record(stream)
        if ev: ev[3].record(stream)
        if not top1_fused:
            moe.combine(layer.y_perm, layer.disp.pos_of, layer.w, out=layer.y)
        if ev: ev[4].record(stream)

    def step():
        """One layer forward exactly as MoEShardLayer runs it (its calls, its buffers)."""
        layer(x, bias)

    def new_events(n, m):
        return [[torch.cuda.Event(enable_timing=True) for _ in range(m)] for _ in range(n)]

    def us(pairs):
        return np.array([a.elapsed_time(b) for a, b in pairs]) * 1e3

    def spread(v):
        return {"median": round(float(np.median(v)), 2), "p10": round(float(np.percentile(v, 10)), 2),
                "p90": round(float(np.percentile(v, 90)), 2)}

    # Cache flush, outside the step's events: 512 MiB (more than L2 and MALL together) written,
    # then read back.  The read pass leaves the caches holding clean lines of the scratch
    # buffer only; after the write alone they would hold dirty lines whose write-back to HBM
    # then runs inside the next step (a cost of the flush, not of the layer; the step time
    # after a write-only flush is reported separately).
    scratch = torch.empty(128 * 1024 * 1024, dtype=torch.float32, device=dev)
    flush_sum = torch.empty((), dtype=torch.float32, device=dev)

    def flush(i, read_back=True):
        scratch.fill_(float(i & 0xff))
        if read_back:
            torch.sum(scratch, dim=0, out=flush_sum)

    # untimed warm-up steps, each after a flush like the timed ones; their step times are kept
    # (events around the step only) to show how the step time settles
    wev = new_events(args.warmup, 2)
    for i in range(args.warmup):
        flush(i)
        wev[i][0].record(stream)
        step()
        wev[i][1].record(stream)
    step_parts(ffn_ev=new_events(1, 2)[0])  # first use of the separate calls (host-side setup)
    torch.cuda.synchronize()
    warm_curve = us(wev) if args.warmup else np.zeros(0)

    # the timed steps: every step starts with cold caches (a flush before it, outside its
    # events); value = tokens over the summed step times.  No event inside a step: each event
    # record leaves the GPU idle for a few microseconds.
    sev = new_events(args.steps, 2)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        flush(i + 1)
        sev[i][0].record(stream)
        step()
        sev[i][1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    step_each = us(sev)

    # the same steps after a write-only flush (dirty lines left in L2 and MALL)
    dev_ = new_events(args.steps, 2)
    for i in range(args.steps):
        flush(i + 1, read_back=False)
        dev_[i][0].record(stream)
        step()
        dev_[i][1].record(stream)
    torch.cuda.synchronize()
    dirty_each = us(dev_)

    # the expert step's own time: as many cold-cache steps again, made of the separate calls
    # with events around the expert-step call (the roofline's kernel time)
    fev = new_events(args.steps, 2)
    torch.cuda.synchronize()
    for i in range(args.steps):
        flush(i + 1)
        step_parts(ffn_ev=fev[i])
    torch.cuda.synchronize()
    ffn_each = us(fev)

    # warm caches: back-to-back steps, wall clock (an extra figure, not the headline)
    warm = None
    if args.warm_steps:
        for _ in range(5):  # untimed: the clock and the caches settle after the host's pause
            step()
        torch.cuda.synchronize()
        tw = time.perf_counter()
        for i in range(args.warm_steps):
            step()
        torch.cuda.synchronize()
        wall_w = time.perf_counter() - tw
        warm = {"steps": args.warm_steps, "tokens_per_s": round(cfg.T * args.warm_steps / wall_w, 1),
                "ms_per_step": round(wall_w / args.warm_steps * 1e3, 4),
                "note": "back-to-back steps without a flush, wall clock; inputs and weights partly in L2/MALL"}

    # stage breakdown from a separate, untimed pass (its events add gaps between calls)
    nbrk = min(args.steps, 10)
    events = new_events(nbrk + 1, 5)
    step_parts(ev=events.pop())  # the separate route and dispatch calls' first use (host-side setup)
    for i in range(nbrk):
        flush(i)
        step_parts(ev=events[i])
    torch.cuda.synchronize()
    del scratch
    stage = np.zeros(4)
    for ev in events:
        for s in range(4):
            stage[s] += ev[s].elapsed_time(ev[s + 1])
    stage_us = stage / nbrk * 1e3

    step_us = float(np.mean(step_each))
    ms_per_step = step_us * 1e-3
    tokens_per_s = cfg.T / (step_us * 1e-6)
    ffn_us = float(np.mean(ffn_each))

    counts = layer.disp.counts.cpu().numpy()
    A, h, f = cfg.A, cfg.h, cfg.f
    n_m = 3 if cfg.act == "swiglu" else 2
    es = 2 if cfg.dtype == "bf16" else 4
    touched = int((counts > 0).sum())
    ffn_flops = 2.0 * n_m * A * h * f
    ffn_bytes = n_m * h * f * es * touched + 2 * A * h * es
    ffn_s = ffn_us * 1e-6
    achieved_gbs = ffn_bytes / ffn_s / 1e9
    achieved_tflops = ffn_flops / ffn_s / 1e12
    peak_tf = PEAK_BF16_TFLOPS if cfg.dtype == "bf16" else PEAK_F32_TFLOPS
    hbm_bound = ffn_bytes / (PEAK_HBM_GBS * 1e9) > ffn_flops / (peak_tf * 1e12)
    roof = ({"bound": "hbm", "achieved": round(achieved_gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
             "frac": round(achieved_gbs / PEAK_HBM_GBS, 4)} if hbm_bound else
            {"bound": "mfma", "achieved": round(achieved_tflops, 1), "peak": peak_tf, "unit": "TFLOP/s",
             "frac": round(achieved_tflops / peak_tf, 4)})
    roof["traffic"] = measured_traffic(args.config)
    roof["kernel"] = ("moe_expert_ffn_shard" + ("_top1" if top1_fused else "" if args.unfused_gather else "_gather") +
                      " (grouped GEMM1+act and GEMM2, one launch each; calls of at most 512 bf16 rows"
                      " add one launch that sums the K parts of GEMM2); HIP events around the call in a "
                      "second pass of as many cold-cache steps as the timed ones, made of the layer's calls "
                      "one by one (the timed steps carry no event inside them)")
    roof["algorithmic"] = {"bytes": ffn_bytes, "flops": ffn_flops, "touched_experts": touched,
                           "mfma_util": round(achieved_tflops / peak_tf, 4),
                           "hbm_frac": round(achieved_gbs / PEAK_HBM_GBS, 4)}

    sb = stage_bytes(cfg, not args.unfused_gather, top1_fused, bias is not None and bias.dim() == 2)
    stages_hbm = {}
    for name, t_us in (("route", stage_us[0]), ("dispatch", stage_us[1]), ("combine", stage_us[3])):
        if sb[name] and t_us > 0:
            gbs = sb[name] / (t_us * 1e-6) / 1e9
            stages_hbm[name] = {"bytes": sb[name], "us": round(t_us, 2), "gbs": round(gbs, 1),
                                "frac": round(gbs / PEAK_HBM_GBS, 4)}
    stages_hbm["note"] = ("algorithmic bytes (inputs read once, outputs written once) over the stage's time in "
                          "the untimed pass (cold caches, events between calls), against 8 TB/s")

    out = {
        "metric": "MoE-layer tokens/sec on 1 MI355X; expert-GEMM MFMA util vs peak",
        "value": round(tokens_per_s, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}: T={cfg.T} h={cfg.h} E={cfg.E} top-{cfg.k} inner {cfg.f} of {cfg.F} "
                               f"({cfg.act}), routing {cfg.routing[0]}",
                   "tokens": cfg.T, "hidden": h, "experts": cfg.E, "top_k": cfg.k, "shard_inner_width": f,
                   "parallelism": "single device"},
        "timing": ("cold caches: 512 MiB written and read back before every timed step, outside HIP events that "
                   "bracket the step (MoEShardLayer.forward, no event inside it); value = tokens / mean step "
                   f"time; wall clock of the timed loop (flushes included) {wall * 1e3:.2f} ms"),
        "after_write_only_flush": {"step_us": spread(dirty_each),
                                   "tokens_per_s": round(cfg.T / (float(np.mean(dirty_each)) * 1e-6), 1),
                                   "note": "the same steps after a flush that writes 512 MiB without reading it "
                                           "back: the write-back of its dirty lines runs inside the step"},
        "stages_us": {"route": round(stage_us[0], 2), "dispatch": round(stage_us[1], 2),
                      "expert_ffn": round(stage_us[2], 2), "combine": round(stage_us[3], 2),
                      "note": "separate untimed pass with events between calls" +
                              ("; top-1: the combine is part of the expert step" if top1_fused else "")},
        "stages_hbm": stages_hbm,
        "expert_ffn_us_timed": round(ffn_us, 2),
        "timed_steps_us": {"step": spread(step_each), "expert_ffn": spread(ffn_each)},
        "warmup_steps_us": {"first": [round(float(v), 1) for v in warm_curve[:5]],
                            "last5_median": round(float(np.median(warm_curve[-5:])), 1) if len(warm_curve) else None},
        "roofline": roof,
    }
    if warm is not None:
        out["warm_cache"] = warm
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(args.config, args.seed)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
