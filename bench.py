"""Benchmark of the MI355X FP8 FFN (one transformer layer's FFN per step).

A step is one call of the whole hot path, lacache_ffn_fp8: fused RMSNorm +
1x128 e4m3 quantization, FP8 gate/up GEMM with fused SwiGLU re-quantization,
FP8 down GEMM to bf16. Inputs are seeded synthetic activations and weights
(LLaDA-8B FFN shapes, H=4096, I=12288), resident in HBM before timing.
Weights rotate over several independently drawn layers, more bytes than the
256 MB Infinity Cache holds, so every step streams its weights from HBM.

Timing: W warm-up steps, then the K steps are captured once in a HIP graph
(as a serving loop runs its decode steps; every step is the whole call). The
graph is replayed untimed for at least half a second; after a device
synchronization (the barrier) a few more untimed replays are queued and the
timed replay of exactly K steps follows them between HIP events, then the
closing synchronization. The replays queued after the barrier keep the GPU
busy while the host submits the timed one: a replay that starts on a GPU left
idle by the barrier runs slower while the clocks come back up, which is
reported as ms_per_step_after_idle. --eager times the plain host loop
instead (its figures are reported either way).

Prints one JSON line. The default workload is the batched long sequence
(8 x 1024 = 8192 tokens, MFMA-bound), the largest single-GPU configuration;
the same line nests the 32-token decode block (HBM-bound), measured in the
same run on its own weights. --workload selects another. For the 31-layer
stack (stack31_m512_h4096_i12288) a step is one denoising step through all 31
layers (all resident in HBM), with the residual adds between them (fused into
the next layer's norm, the last one a plain add); 32 steps by default, one per
denoising step, each on its own input. Besides the whole-step throughput the
line carries the dominant kernel's roofline figures (timed live with HIP
events around graph-captured back-to-back calls of its stage alone, and
compared with the same kernel's average in the committed rocprofv3 trace) and
the CPU oracle's throughput on a bounded sample of the same workload.

  python bench.py [--gpus 1] [--steps 50] [--warmup 10] [--workload batch8x1024_h4096_i12288]
"""

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "FP8 FFN TFLOP/s + tokens/s per layer (H=4096,I=12288); % FP8 MFMA / HBM peak"
PEAK_HBM_GBPS = 8000.0
PEAK_FP8_TFLOPS = 5033.0  # dense FP8 MFMA: 256 CU x 2.4 GHz x 8192 FLOP/clk
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "pmc_traffic.json")
KERNEL_SOURCES = {  # the files that define each kernel and its launch (item order, limits)
    "gateup_skinny": ["gemm_skinny.hip", "device.h", "launch.h"],
    "hquant_skinny": ["gemm_skinny.hip", "device.h", "launch.h"],
    "down_skinny": ["gemm_skinny.hip", "device.h", "launch.h"],
    "reduce_tiled": ["gemm_tiled.hip", "device.h", "launch.h"],
    "gateup_tiled": ["gemm_tiled.hip", "device.h", "launch.h"],
    "down_tiled": ["gemm_tiled.hip", "device.h", "launch.h"],
}


def parse(argv=None):
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=None,
                   help="timed steps (default 50; 32 for the stack, one step per denoising step)")
    p.add_argument("--warmup", type=int, default=10)
    p.add_argument("--workload", default=DEFAULT_WORKLOAD,
                   help="an FFN workload, an attention workload (attn_*: the first-layer FACache attention), or "
                        "first_layer_n512 (the token-wise first layer with EmbedCache / RoPECache)")
    p.add_argument("--weight-sets", type=int, default=4)
    p.add_argument("--granularity", action="store_true",
                   help="time the FFN at the three quantization granularities (per group, per token, per tensor) "
                        "and report each one's error against the unquantized bf16 FFN")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-nested", action="store_true",
                   help="with the default workload, skip the nested 32-token decode-block measurement")
    p.add_argument("--eager", action="store_true",
                   help="time the eager host loop instead of the HIP-graph replay of the K steps")
    p.add_argument("--profile-only", action="store_true",
                   help="run warmup + timed steps only (for rocprofv3), print the line without the CPU leg")
    p.add_argument("--warm-s", type=float, default=WARM_S,
                   help="seconds of untimed graph replays before the timed one (shorter under a profiler)")
    p.add_argument("--calibrate-copy", action="store_true",
                   help="also run a plain device copy of 256 MiB three times (the HBM counter calibration)")
    p.add_argument("--counters-from", nargs=2, metavar=("COUNTER_CSV", "KERNEL_TRACE_CSV"),
                   help="summarize a rocprofv3 --pmc counter CSV per kernel (averages per dispatch; MFMA busy "
                        "fraction of the SIMDs' active cycles, FP8 MFMA FLOP from the MOPS counter, against the "
                        "kernel durations of a --kernel-trace CSV of the same command), then exit")
    p.add_argument("--traffic-from", nargs=3, metavar=("FETCH_CSV", "WRITE_CSV", "WORKLOAD"),
                   help="turn two rocprofv3 --pmc counter CSVs (FETCH_SIZE, WRITE_SIZE) of a --calibrate-copy "
                        "run into per-launch HBM bytes in profiles/pmc_traffic.json, then exit")
    args = p.parse_args(argv)
    if args.steps is None:
        args.steps = 32 if args.workload.startswith("stack") else 50
    return args


def code_hash(texts):
    """Hash of C++/HIP source texts with comments and blank space removed."""
    h = hashlib.sha256()
    for t in texts:
        t = re.sub(r"/\*.*?\*/", "", t, flags=re.S)
        t = re.sub(r"//[^\n]*", "", t)
        h.update("\n".join(ln.strip() for ln in t.splitlines() if ln.strip()).encode())
    return h.hexdigest()[:16]


def source_sha(kernel):
    """Hash of the kernel's sources without comments: counter data stay
    attached to the code they were taken on, and only a change of code (not
    of its comments) detaches them."""
    texts = []
    for f in KERNEL_SOURCES[kernel]:
        with open(os.path.join(ROOT, "paper_2607_16339_amd", "csrc", f), encoding="utf-8") as fh:
            texts.append(fh.read())
    return code_hash(texts)


def stage_bytes(M, H, I):
    """Algorithmic HBM bytes per launch of each stage (each operand read once,
    each result written once)."""
    g = 128
    return {
        "norm": 2 * M * H + 2 * H + M * H + 4 * M * H // g,
        "gateup": 2 * I * H + 4 * (2 * I // g) * (H // g) + M * H + 4 * M * H // g + M * I + 4 * M * I // g,
        "down": H * I + 4 * (H // g) * (I // g) + M * I + 4 * M * I // g + 2 * M * H,
        # the skinny gate/up's weight-streaming kernel alone: its inputs and
        # its fp32 h (which the h-quantization kernel then reads)
        "gateup_stream": 2 * I * H + 4 * (2 * I // g) * (H // g) + M * H + 4 * M * H // g + 4 * M * I,
    }


COPY_BYTES = 256 << 20
WARM_S = 0.5  # seconds of untimed graph replays before the timed one
DEFAULT_WORKLOAD = "batch8x1024_h4096_i12288"  # MFMA-bound: 8 sequences x 1024 tokens
NESTED_WORKLOAD = "block32_h4096_i12288"  # HBM-bound: one 32-token decode block
# the skinny gate/up stage ends with a separate h-quantization kernel
SKINNY_HQUANT_KERNEL = True


def kernel_key(name):
    """Short kernel key of a rocprofv3 kernel name."""
    if "skinny_gateup_kernel" in name:
        return "gateup_skinny"
    if "skinny_down_kernel" in name:
        return "down_skinny"
    if "skinny_hquant" in name:
        return "hquant_skinny"
    if "split_reduce" in name:
        return "reduce_tiled"
    if "gemm_tiled_kernel<true" in name:
        return "gateup_tiled"
    if "gemm_tiled_kernel<false" in name:
        return "down_tiled"
    if "rmsnorm_quant" in name:
        return "rmsnorm_quant"
    if "copyBuffer" in name:
        return "copy"
    return None


CUS = 256
SIMDS_PER_CU = 4


def counters_from(counter_csv, trace_csv):
    """Per-kernel averages of a rocprofv3 --pmc run (values summed over a
    dispatch's rows, then averaged over the kernel's dispatches), with
      mfma_busy_frac   = SQ_VALU_MFMA_BUSY_CYCLES / (4 SIMDs x SQ_BUSY_CU_CYCLES)
      fp8_flop         = 512 x SQ_INSTS_VALU_MFMA_MOPS_F8 per dispatch
      fp8_frac_of_peak = fp8_flop / (average duration in the kernel trace) / peak
      implied_clock_ghz = the clock at which that busy share gives that rate
                          (a 16x16x128 FP8 MFMA keeps a SIMD busy 32 cycles:
                          2048 FLOP per SIMD per cycle)
    The kernel trace is a separate --kernel-trace run of the same command
    (counter collection serializes kernels and would lengthen them)."""
    import csv
    import collections

    per = collections.defaultdict(lambda: collections.defaultdict(float))
    names, res = {}, {}
    for r in csv.DictReader(open(counter_csv)):
        d = r["Dispatch_Id"]
        per[d][r["Counter_Name"]] += float(r["Counter_Value"])
        names[d] = r["Kernel_Name"]
        res[d] = {c: int(r[c]) for c in ("VGPR_Count", "Accum_VGPR_Count", "SGPR_Count", "LDS_Block_Size",
                                         "Scratch_Size", "Workgroup_Size", "Grid_Size") if r.get(c, "").isdigit()}
    agg = collections.defaultdict(lambda: collections.defaultdict(list))
    kres = {}
    for d, cs in per.items():
        k = kernel_key(names[d])
        if k is None:
            continue
        kres[k] = res[d]
        for c, v in cs.items():
            agg[k][c].append(v)
    dur = collections.defaultdict(list)
    for r in csv.DictReader(open(trace_csv)):
        k = kernel_key(r["Kernel_Name"])
        if k is not None:
            dur[k].append((float(r["End_Timestamp"]) - float(r["Start_Timestamp"])) * 1e-9)
    out = {}
    for k, cs in agg.items():
        a = {c: sum(v) / len(v) for c, v in cs.items()}
        e = {"dispatches": len(next(iter(cs.values()))), "avg": {c: round(v, 1) for c, v in sorted(a.items())},
             "resources": kres.get(k, {})}
        if "SQ_VALU_MFMA_BUSY_CYCLES" in a and a.get("SQ_BUSY_CU_CYCLES"):
            # both counters summed over the CUs, in the same clock: the MFMA
            # pipes' busy share of the cycles the CUs were busy
            e["mfma_busy_frac"] = round(a["SQ_VALU_MFMA_BUSY_CYCLES"] / (SIMDS_PER_CU * a["SQ_BUSY_CU_CYCLES"]), 4)
        if "SQ_INSTS_VALU_MFMA_MOPS_F8" in a:
            e["fp8_flop"] = 512.0 * a["SQ_INSTS_VALU_MFMA_MOPS_F8"]
            if dur.get(k):
                t = sum(dur[k]) / len(dur[k])
                e["trace_avg_us"] = round(t * 1e6, 2)
                e["fp8_frac_of_peak"] = round(e["fp8_flop"] / t / 1e12 / PEAK_FP8_TFLOPS, 4)
                if e.get("mfma_busy_frac"):
                    # FLOP rate = busy share x SIMDs x 2048 FLOP/clk x clock: the clock it implies
                    e["implied_clock_ghz"] = round(e["fp8_flop"] / t / (e["mfma_busy_frac"] * CUS * SIMDS_PER_CU * 2048)
                                                   / 1e9, 3)
        out[k] = e
    print(json.dumps(out, indent=1, sort_keys=True))


def traffic_from(fetch_csv, write_csv, workload):
    """Per-dispatch FETCH_SIZE / WRITE_SIZE (KiB) averaged per kernel, scaled by
    the ratio of the known bytes of a plain 256 MiB device copy to what the
    same counter reads for that copy."""
    import csv
    import collections

    def per_kernel(path, counter):
        per = collections.defaultdict(float)
        names = {}
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] != counter:
                continue
            d = r["Dispatch_Id"]
            per[d] += float(r["Counter_Value"])
            names[d] = r["Kernel_Name"]
        out = collections.defaultdict(list)
        for d, v in per.items():
            k = kernel_key(names[d])
            if k:
                out[k].append(v * 1024.0)  # KiB -> bytes
        # the runtime's own small copies share the copy kernel: keep the 256 MiB ones
        big = max(out["copy"])
        out["copy"] = [v for v in out["copy"] if v > big / 2]
        return {k: sum(v) / len(v) for k, v in out.items()}

    fetch = per_kernel(fetch_csv, "FETCH_SIZE")
    write = per_kernel(write_csv, "WRITE_SIZE")
    f_scale = COPY_BYTES / fetch["copy"]
    w_scale = COPY_BYTES / write["copy"]
    try:
        with open(TRAFFIC_FILE) as f:
            table = json.load(f)
    except (OSError, ValueError):
        table = {}
    for k in KERNEL_SOURCES:
        if k in fetch and k in write:
            table[k + ":" + workload] = {
                "fetch_bytes": round(fetch[k] * f_scale), "write_bytes": round(write[k] * w_scale),
                "hbm_bytes_per_launch": round(fetch[k] * f_scale + write[k] * w_scale),
                "copy_scale": {"fetch": round(f_scale, 4), "write": round(w_scale, 4)},
                "source_sha": source_sha(k)}
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(table, f, indent=1, sort_keys=True)
    print(json.dumps({k: v for k, v in table.items() if k.endswith(":" + workload)}, indent=1))


def main():
    args = parse()
    if args.traffic_from:
        traffic_from(*args.traffic_from)
        return
    if args.counters_from:
        counters_from(*args.counters_from)
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path (the FFN shards by rows with no "
              "exchange). Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2607_16339_amd as lc
    import synth

    if args.workload.startswith("attn_"):
        attention_main(args)
        return
    if args.granularity:
        granularity_main(args)
        return
    if args.workload.startswith("first_layer"):
        first_layer_main(args)
        return
    w = synth.WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    lc.lib()  # fails loudly when the HIP library is missing
    line = ffn_line(args, w, dev)
    if args.workload == DEFAULT_WORKLOAD and not args.no_nested:
        # the HBM-bound decode block, measured in the same run (its own weights)
        w2 = synth.WORKLOADS[NESTED_WORKLOAD]
        nested = ffn_line(args, w2, dev, nested=True)
        keep = ("value", "unit", "ms_per_step", "tokens_per_s", "hbm_GBps_min_bytes", "frac_hbm_peak",
                "frac_fp8_peak", "ms_per_step_after_idle", "ms_per_step_graph_replays", "stage_ms", "roofline",
                "vs_bf16_ffn", "cpu_baseline", "config", "steps")
        line["nested"] = {NESTED_WORKLOAD: {k: nested[k] for k in keep if k in nested}}
    print(json.dumps(line), flush=True)


def dev_bf16_fn(dev):
    import numpy as np
    import torch

    def dev_bf16(bits):
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16).copy()).view(torch.bfloat16).to(dev)
    return dev_bf16


def ffn_weight_sets(w, n, dev):
    """n independently drawn layers of the workload's weights, quantized on
    the GPU (bf16 copies freed), each with its own input x; the seeded bf16
    draws run on host threads (the generator releases the GIL)."""
    from concurrent.futures import ThreadPoolExecutor

    import numpy as np

    import paper_2607_16339_amd as lc
    import synth
    dev_bf16 = dev_bf16_fn(dev)
    with ThreadPoolExecutor(max_workers=min(4, n)) as ex:
        futs = [ex.submit(lambda layer: (synth.make_weights(w, layer), synth.make_x(w, layer=layer, step=layer - 1)),
                          layer) for layer in range(1, n + 1)]
        sets = []
        for f in futs:
            b, xb = f.result()
            wgu = dev_bf16(np.concatenate([b["w_gate"], b["w_up"]], axis=0))
            wgu_q, wgu_s = lc.quantize_weights(wgu)
            del wgu
            wd = dev_bf16(b["w_down"])
            wd_q, wd_s = lc.quantize_weights(wd)
            del wd
            sets.append(dict(norm_w=dev_bf16(b["norm_w"]), wgu_q=wgu_q, wgu_s=wgu_s, wd_q=wd_q, wd_s=wd_s,
                             x=dev_bf16(xb)))
            del b
    return sets


def time_graph(g, K, stream, warm_s=WARM_S, min_warm=3):
    """Times one replay of a captured graph of K steps. Untimed replays run
    back to back for at least warm_s seconds first; after the barrier
    (device synchronization) a few more untimed replays are queued, then the
    timed replay between HIP events, then the closing synchronization. The
    replays queued after the barrier keep the GPU busy while the host submits
    the timed replay: a timed replay that starts on an idle GPU (measured too,
    as ms_after_idle) runs slower while the clocks come back up. Returns a
    dict of per-step milliseconds."""
    import torch
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    g.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    est_s = max(e0.elapsed_time(e1) * 1e-3, 1e-6)
    n_warm = max(min_warm, min(5000, int(warm_s / est_s) + 1))
    for _ in range(n_warm):
        g.replay()
    torch.cuda.synchronize()
    # diagnostic: a replay that starts right after the barrier, on an idle GPU
    e0.record(stream)
    g.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    after_idle = e0.elapsed_time(e1) / K
    # the timed replay: barrier, untimed replays covering >= 5 ms of GPU time,
    # then exactly one timed replay of the K steps
    torch.cuda.synchronize()
    n_pre = max(2, int(5e-3 / est_s) + 1)
    t_wall = time.perf_counter()
    for _ in range(n_pre):
        g.replay()
    e0.record(stream)
    t_sub = time.perf_counter()
    g.replay()  # the timed region: exactly K steps
    t_sub = time.perf_counter() - t_sub
    e1.record(stream)
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall
    timed = e0.elapsed_time(e1) / K
    more = []
    for _ in range(5):
        e0.record(stream)
        g.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        more.append(e0.elapsed_time(e1) / K)
    return {"timed": timed, "after_idle": after_idle, "more": more, "submit_ms": t_sub * 1e3,
            "n_pre": n_pre, "wall_s": t_wall}


def trace_kernel_us(workload, name_prefix):
    """Average duration (us) of a kernel in the committed rocprofv3 kernel
    trace summary of the workload (profiles/kernel_trace_ffn_<workload>.txt),
    or None."""
    path = os.path.join(ROOT, "profiles", "kernel_trace_ffn_%s.txt" % workload)
    try:
        with open(path) as f:
            for ln in f:
                if ln.startswith(name_prefix):
                    cols = ln[74:].split()
                    return float(cols[1])
    except (OSError, ValueError, IndexError):
        return None
    return None


def ffn_line(args, w, dev, nested=False):
    """The bench line of one FFN workload (see the module docstring)."""
    import numpy as np
    import torch

    import paper_2607_16339_amd as lc
    import synth

    M, H, I = w.M, w.H, w.I
    dev_bf16 = dev_bf16_fn(dev)
    L = w.layers
    if w.act == "stack":
        # ---- the stack: one step is one denoising step through all L layers.
        # Layer 1 runs the plain FFN on the step's input; layers 2..L add the
        # previous layer's output into the residual stream inside their norm
        # (AddNorm); the last output is added at the end.
        layers = stack_weights(w, dev_bf16)
        xin = [dev_bf16(synth.make_x(w, layer=1, step=t)) for t in range(w.steps)]
        resid = torch.empty((M, H), dtype=torch.bfloat16, device=dev)
        outs = [torch.empty((M, H), dtype=torch.bfloat16, device=dev) for _ in range(2)]

        def step(i):
            resid.copy_(xin[i % len(xin)])
            a = layers[0]
            lc.lacache_ffn_fp8(resid, a["norm_w"], a["wgu_q"], a["wgu_s"], a["wd_q"], a["wd_s"], outs[0])
            for layer in range(1, L):
                a = layers[layer]
                lc.lacache_ffn_fp8_addnorm(resid, outs[(layer - 1) % 2], a["norm_w"], a["wgu_q"], a["wgu_s"],
                                           a["wd_q"], a["wd_s"], outs[layer % 2])
            lc.lacache_add_bf16(resid, outs[(L - 1) % 2])

        probe = resid
        out = outs[0]
        # the stage timings below use the first layers on the first steps' inputs
        sets = [dict(layers[i], x=xin[i]) for i in range(min(args.weight_sets, L))]
    else:
        sets = ffn_weight_sets(w, args.weight_sets, dev)
        out = torch.empty((M, H), dtype=torch.bfloat16, device=dev)

        def step(i):
            s = sets[i % len(sets)]
            lc.lacache_ffn_fp8(s["x"], s["norm_w"], s["wgu_q"], s["wgu_s"], s["wd_q"], s["wd_s"], out)

        probe = out
    torch.cuda.synchronize()
    S = len(sets)
    K = args.steps if not (nested and w.act == "stack") else args.steps

    stream = torch.cuda.current_stream()
    # eager: one host call per step, per-step events
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(K + 1)]
    ev[0].record(stream)
    for i in range(K):
        step(i)
        ev[i + 1].record(stream)
    torch.cuda.synchronize()
    ms_eager = ev[0].elapsed_time(ev[-1]) / K
    per_step = np.array([ev[i].elapsed_time(ev[i + 1]) for i in range(K)])
    pct = {"p10": float(np.percentile(per_step, 10)), "p50": float(np.percentile(per_step, 50)),
           "p90": float(np.percentile(per_step, 90))}

    # graph: the K steps captured once in a HIP graph (as a serving loop runs
    # its decode steps), every step the whole call on its own weight set
    tg = None
    if not args.eager:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for i in range(K):
                step(i)
        # the replay must reproduce the eager result of the same step
        g.replay()
        torch.cuda.synchronize()
        got = probe.clone()
        step(K - 1)
        torch.cuda.synchronize()
        if not torch.equal(got, probe):
            raise RuntimeError("graph replay of the FFN step differs from the eager call")
        tg = time_graph(g, K, stream, warm_s=args.warm_s)
        del g
        ms = tg["timed"]
        t_wall = tg["wall_s"]
    else:
        ms = ms_eager
        t_wall = float(per_step.sum()) * 1e-3
    if args.calibrate_copy and not nested:
        src = torch.empty(COPY_BYTES, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    flop = 6.0 * M * H * I * L
    tflops = flop / (ms * 1e-3) / 1e12
    tok_s = M / (ms * 1e-3)
    bytes_min = (3 * H * I + 4 * (3 * I // 128) * (H // 128) + 2 * H + 4 * M * H) * L
    gbps = bytes_min / (ms * 1e-3) / 1e9

    k_ms, roof = stage_timings(args, w, sets, out, dev)
    roof["step_frac"] = round(tflops / PEAK_FP8_TFLOPS if roof["bound"] == "mfma" else gbps / PEAK_HBM_GBPS, 4)

    line = {
        "metric": METRIC, "value": round(tflops, 3), "unit": "TFLOP/s", "n_gpus": 1, "steps": K,
        "warmup": args.warmup, "ms_per_step": round(ms, 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "fp8_e4m3 (fp32 accumulate)", "data": "synthetic",
        "config": {"workload": w.name, "M": M, "H": H, "I": I, "group": 128,
                   "weight_sets": L if w.act == "stack" else S, "path": "skinny" if M <= 64 else "tiled",
                   "layers": L},
        "tokens_per_s": round(tok_s, 1), "hbm_GBps_min_bytes": round(gbps, 1),
        "frac_hbm_peak": round(gbps / PEAK_HBM_GBPS, 4), "frac_fp8_peak": round(tflops / PEAK_FP8_TFLOPS, 4),
        "step_timing": "HIP graph replay of the K steps" if tg is not None else "eager host loop",
        "ms_per_step_eager": round(ms_eager, 5),
        "ms_per_step_eager_pct": {k: round(v, 5) for k, v in pct.items()},
        "stage_ms": {k: round(v, 5) for k, v in k_ms.items()}, "stage_timing": "HIP graph of back-to-back stage calls",
        "wall_s_timed": round(t_wall, 4),
        "roofline": roof,
    }
    if tg is not None:
        line["ms_per_step_graph_replays"] = [round(v, 5) for v in tg["more"]]
        line["ms_per_step_after_idle"] = round(tg["after_idle"], 5)
        line["replay_submit_ms"] = round(tg["submit_ms"], 4)
        line["replays_queued_before_timed"] = tg["n_pre"]
    if not args.profile_only:
        line["vs_bf16_ffn"] = error_vs_bf16(w, sets[0], out, dev)
    if not args.no_cpu_baseline and not args.profile_only:
        line["cpu_baseline"] = cpu_baseline(w, sets, out, dev)
    del sets
    torch.cuda.synchronize()
    return line


def stage_timings(args, w, sets, out, dev):
    """Each stage timed alone: the stage entry points launch the same kernels
    as the fused call. R back-to-back calls (rotating over the weight sets)
    are captured in a HIP graph, so that the host's per-call cost does not
    leave the GPU idle between them; the graph is replayed between HIP events
    on the stream it runs on. Returns (stage ms, roofline of the dominant
    kernel)."""
    import torch

    import paper_2607_16339_amd as lc

    M, H, I = w.M, w.H, w.I
    S = len(sets)
    skinny = M <= 64
    xq = torch.empty((M, H), dtype=torch.uint8, device=dev)
    xs = torch.empty((H // 128, M), dtype=torch.float32, device=dev)
    hq = torch.empty((M, I), dtype=torch.uint8, device=dev)
    hs = torch.empty((I // 128, M), dtype=torch.float32, device=dev)
    sb = stage_bytes(M, H, I)
    stage_fn = {
        "norm": lambda s: lc.lacache_rmsnorm_quant(s["x"], s["norm_w"], xq, xs),
        "gateup": lambda s: lc.lacache_gateup_swiglu_quant(xq, xs, s["wgu_q"], s["wgu_s"], hq, hs),
        "down": lambda s: lc.lacache_down_proj(hq, hs, s["wd_q"], s["wd_s"], out),
    }
    names = ["norm", "gateup", "down"]
    # at M <= 32 the skinny gate/up stage ends with the h-quantization kernel
    # that lacache_quant_rows_g launches alone (33..64 rows: a variant that
    # also adds the two K halves)
    split_stage = skinny and M <= 32 and SKINNY_HQUANT_KERNEL
    if split_stage:
        # the h-quantization kernel of the skinny gate/up stage, timed alone:
        # the same kernel on the same sizes (lacache_quant_rows_g at group
        # granularity) over the real h of the workload
        hbuf = torch.empty((M, I), dtype=torch.float32, device=dev)
        lc.lacache_rmsnorm_quant(sets[0]["x"], sets[0]["norm_w"], xq, xs)
        lc.lacache_gateup_swiglu_quant(xq, xs, sets[0]["wgu_q"], sets[0]["wgu_s"], hq, hs, hbuf)
        hq2 = torch.empty((M, I), dtype=torch.uint8, device=dev)
        hs2 = torch.empty((I // 128, M), dtype=torch.float32, device=dev)
        stage_fn["hquant"] = lambda s: lc.lacache_quant_rows_g(hbuf, hq2, hs2, None, lc.LACACHE_GRAN_GROUP)
        names.append("hquant")
    reps = max(min(args.steps, 64), 8)
    k_ms = {}
    for name in names:
        fn = stage_fn[name]
        for i in range(S):  # inputs of every stage valid, workspace allocated
            for n2 in ("norm", "gateup", "down"):
                stage_fn[n2](sets[i])
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for i in range(reps):
                fn(sets[i % S])
        g.replay()
        torch.cuda.synchronize()
        # the replay must reproduce the eager result of its last call
        probe = {"norm": xq, "gateup": hq, "down": out, "hquant": hq2 if split_stage else None}[name]
        got = probe.clone()
        fn(sets[(reps - 1) % S])
        torch.cuda.synchronize()
        if not torch.equal(got, probe):
            raise RuntimeError("graph replay of the %s stage differs from the eager call" % name)
        t = time_graph(g, reps, torch.cuda.current_stream(), warm_s=min(0.1, args.warm_s), min_warm=2)
        k_ms[name] = t["timed"]
        del g
    dom = "gateup"
    if split_stage:
        # The skinny gate/up stage is the weight-streaming kernel followed by
        # the small h-quantization kernel. The dominant kernel is the first:
        # its time is the stage's minus the h-quantization kernel's, both timed
        # live above; the stage's own figure is reported beside it.
        kparts = ["gateup_skinny"]
        k_stream = k_ms[dom] - k_ms["hquant"]
        achieved = sb["gateup_stream"] / (k_stream * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                "frac": round(achieved / PEAK_HBM_GBPS, 4)}
        roof["kernel"] = "gateup_skinny (the weight stream)"
        roof["kernel_ms"] = round(k_stream, 5)
        roof["kernel_ms_from"] = "gate/up stage minus the h-quantization kernel timed alone"
        roof["algorithmic_bytes"] = sb["gateup_stream"]
        st_ach = sb[dom] / (k_ms[dom] * 1e-3) / 1e9
        roof["stage"] = {"kernels": "gateup_skinny + hquant_skinny", "ms": round(k_ms[dom], 5),
                         "algorithmic_bytes": sb[dom], "achieved": round(st_ach, 1),
                         "frac": round(st_ach / PEAK_HBM_GBPS, 4)}
        trace_prefix = "void lacache::(anonymous namespace)::skinny_gateup_kernel"
        per_byte = sb["gateup_stream"]
    elif skinny:
        kparts = ["gateup_skinny"] + (["hquant_skinny"] if SKINNY_HQUANT_KERNEL else [])
        achieved = sb[dom] / (k_ms[dom] * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                "frac": round(achieved / PEAK_HBM_GBPS, 4)}
        roof["kernel"] = "gateup_skinny" + (" + hquant_skinny (the stage)" if SKINNY_HQUANT_KERNEL else "")
        roof["kernel_ms"] = round(k_ms[dom], 5)
        roof["algorithmic_bytes"] = sb[dom]
        trace_prefix = "void lacache::(anonymous namespace)::skinny_gateup_kernel"
        per_byte = sb[dom]
    else:
        kparts = ["gateup_tiled"]
        achieved = 4.0 * M * H * I / (k_ms[dom] * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 1), "peak": PEAK_FP8_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / PEAK_FP8_TFLOPS, 4)}
        roof["kernel"] = "gateup_tiled"
        roof["kernel_ms"] = round(k_ms[dom], 5)
        roof["algorithmic_flop"] = 4 * M * H * I
        trace_prefix = "void lacache::gemm_tiled_kernel<true"
        per_byte = None
    roof["kernel_ms_timing"] = "HIP events around a graph of back-to-back calls of the stage alone"
    # the same kernel's average duration in the committed rocprofv3 trace
    us = trace_kernel_us(w.name, trace_prefix)
    if us is not None:
        tr = (per_byte / (us * 1e-6) / 1e9 / PEAK_HBM_GBPS) if per_byte else (
            4.0 * M * H * I / (us * 1e-6) / 1e12 / PEAK_FP8_TFLOPS)
        roof["trace"] = {"file": "profiles/kernel_trace_ffn_%s.txt" % w.name, "avg_us": us,
                         "frac": round(tr, 4), "live_vs_trace": round(roof["kernel_ms"] * 1e3 / us - 1, 4)}
    roof["traffic"] = None
    try:
        with open(TRAFFIC_FILE) as f:
            table = json.load(f)
        parts = [table.get(k + ":" + w.name) for k in kparts]
        if all(t and t.get("source_sha") == source_sha(k) for t, k in zip(parts, kparts)):
            roof["traffic"] = sum(t["hbm_bytes_per_launch"] for t in parts)
    except (OSError, ValueError):
        pass
    return k_ms, roof


def stack_weights(w, dev_bf16):
    """The FP8 weights of the stack's layers 1..L: each layer's seeded bf16
    weights drawn on host threads (the generator releases the GIL), then
    quantized on the GPU; the host and bf16 device copies are freed."""
    from concurrent.futures import ThreadPoolExecutor, as_completed

    import numpy as np

    import paper_2607_16339_amd as lc
    import synth

    layers = [None] * w.layers
    with ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        futs = {ex.submit(synth.make_weights, w, layer): layer for layer in range(1, w.layers + 1)}
        for f in as_completed(futs):
            b = f.result()
            wgu = dev_bf16(np.concatenate([b["w_gate"], b["w_up"]], axis=0))
            wgu_q, wgu_s = lc.quantize_weights(wgu)
            del wgu
            wd = dev_bf16(b["w_down"])
            wd_q, wd_s = lc.quantize_weights(wd)
            del wd
            layers[futs[f] - 1] = dict(norm_w=dev_bf16(b["norm_w"]), wgu_q=wgu_q, wgu_s=wgu_s, wd_q=wd_q,
                                       wd_s=wd_s)
            del b
    return layers


def error_vs_bf16(w, s, out, dev, rows=8):
    """Context figure: the FP8 FFN's output against an unquantized FFN (bf16
    operands, fp64 arithmetic) on the first rows of weight set 1."""
    import numpy as np
    import torch
    import oracle.ffn as O
    import synth

    import paper_2607_16339_amd as lc
    lc.lacache_ffn_fp8(s["x"], s["norm_w"], s["wgu_q"], s["wgu_s"], s["wd_q"], s["wd_s"], out)
    got = out[:rows].float().cpu().numpy().astype(np.float64)
    b = synth.make_weights(w, 1)
    xb = synth.make_x(w, layer=1, step=0)[:rows]
    ref = O.ffn_bf16_reference(xb, b["norm_w"], b["w_gate"], b["w_up"], b["w_down"])
    err = np.abs(got - ref)
    return {"rows": rows, "max_abs_err": float(err.max()), "ref_max_abs": float(np.abs(ref).max()),
            "max_err_rel_to_max": float(err.max() / np.abs(ref).max()),
            "rms_err_rel_to_rms": float(np.sqrt((err ** 2).mean() / (ref ** 2).mean()))}


def cpu_baseline(w, sets, out, dev):
    """The oracle, as it stands (NumPy fp64, BLAS-threaded matmuls), on a
    bounded sample of the same workload: whole-layer calls on up to 512 of
    its rows (the FFN is row-independent), repeated over the weight sets until
    about 10 s of CPU work. Larger workloads are extrapolated from the sample
    and labelled so: M / 512 times the per-call time for the batched
    workload, and L layers x steps for the stack."""
    import numpy as np
    import torch

    import oracle.ffn as O
    import paper_2607_16339_amd as lc
    import synth

    blas = _threads()
    rows = min(w.M, 512)
    t = 0.0
    calls = 0
    while calls < 1 or (t < 10.0 and calls < 64):
        s = sets[calls % len(sets)]
        xb = synth.make_x(w, layer=calls % len(sets) + 1, step=calls % len(sets))[:rows]
        host = [lc.weight_codes_rowmajor(s["wgu_q"]), s["wgu_s"].cpu().numpy(), lc.weight_codes_rowmajor(s["wd_q"]),
                s["wd_s"].cpu().numpy()]
        norm_w = s["norm_w"].view(torch.int16).cpu().numpy().view(np.uint16)
        t0 = time.perf_counter()
        O.ffn(xb, norm_w, host[0], host[1], host[2], host[3], w.I)
        t += time.perf_counter() - t0
        calls += 1
    per_call = t / calls
    flop = 6.0 * rows * w.H * w.I * calls
    r = {"value": round(flop / t / 1e12, 6), "unit": "TFLOP/s", "cores": blas, "kind": "oracle",
         "os_cpu_count": os.cpu_count(), "blas_threads": blas,
         "sample": "%d whole-layer oracle calls on %d of the %d rows (one layer each; the FFN is row-independent): "
                   "%.2f s" % (calls, rows, w.M, t),
         "tokens_per_s_per_layer": round(rows * calls / t, 3), "s_per_sample_call": round(per_call, 4)}
    if rows < w.M or w.layers > 1:
        factor = (w.M / rows) * w.layers
        r["extrapolated"] = {
            "label": "EXTRAPOLATED, not measured: the sample's per-call time x %g" % factor,
            "factor": factor,
            "what": ("one call on all %d rows = %d sample calls of %d rows" % (w.M, w.M // rows, rows))
            if w.layers == 1 else ("one denoising step = %d layers; the whole run of %d steps = x%d"
                                   % (w.layers, w.steps, w.layers * w.steps)),
            "s_per_step": round(per_call * factor, 3)}
        if w.layers > 1:
            r["extrapolated"]["s_whole_run"] = round(per_call * w.layers * w.steps, 2)
    return r


def granularity_main(args):
    """One line for the quantization granularities of the FFN (the paper's
    per-group scheme against per-token and per-tensor, Table
    fp8-granularities): a step is one whole FFN call at the headline
    granularity (per token), timed as a HIP graph of back-to-back calls beside
    the other two; each granularity's error against the unquantized bf16 FFN
    (bf16 operands, fp64 arithmetic) on the first rows of the workload."""
    import numpy as np
    import torch

    import oracle.ffn as O
    import paper_2607_16339_amd as lc
    import synth
    from oracle.bf16 import bf16_to_f32

    w = synth.WORKLOADS[args.workload]
    M, H, I = w.M, w.H, w.I
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    lc.lib()

    def dev_bf16(bits):
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16).copy()).view(torch.bfloat16).to(dev)

    grans = {"group": lc.LACACHE_GRAN_GROUP, "token": lc.LACACHE_GRAN_TOKEN, "tensor": lc.LACACHE_GRAN_TENSOR}
    # the weights of several layers per granularity, more bytes than the
    # Infinity Cache holds, so that every call streams its weights from HBM
    S = args.weight_sets
    sets = {name: [] for name in grans}
    for layer in range(1, S + 1):
        b = synth.make_weights(w, layer)
        wgu = dev_bf16(np.concatenate([b["w_gate"], b["w_up"]], axis=0))
        wd = dev_bf16(b["w_down"])
        for name, g in grans.items():
            sets[name].append(lc.quantize_weights_g(wgu, g) + lc.quantize_weights_g(wd, g))
        del wgu, wd
    b = synth.make_weights(w, 1)
    x = dev_bf16(synth.make_x(w, layer=1, step=0))
    norm_w = dev_bf16(b["norm_w"])
    out = torch.empty((M, H), dtype=torch.bfloat16, device=dev)

    def call(name, i=0):
        gq, gs, gr, dq, ds, dr = sets[name][i % S]
        lc.lacache_ffn_fp8_g(x, norm_w, gq, gs, gr, dq, ds, dr, out, grans[name])

    stream = torch.cuda.current_stream()
    reps = max(min(args.steps, 64), 8)
    ms, gate_ms, errs = {}, {}, {}
    rows = min(M, 8)
    ref = O.ffn_bf16_reference(synth.make_x(w, layer=1, step=0)[:rows], b["norm_w"], b["w_gate"], b["w_up"],
                               b["w_down"])
    for name in grans:
        for _ in range(args.warmup):
            call(name)
        torch.cuda.synchronize()
        got = bf16_to_f32(out[:rows].contiguous().view(torch.int16).cpu().numpy().view(np.uint16)).astype(np.float64)
        errs[name] = {"rms_err_rel_to_rms": float(np.sqrt(((got - ref) ** 2).mean() / (ref ** 2).mean())),
                      "max_err_rel_to_max": float(np.abs(got - ref).max() / np.abs(ref).max())}
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for i in range(reps):
                call(name, i)
        g.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(3):
            g.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        ms[name] = e0.elapsed_time(e1) / (3 * reps)
        del g
    # the dominant kernel of the coarse path: gate/up + SwiGLU writing fp32 h
    gq, gs, gr = sets["token"][0][:3]
    xq = torch.empty((M, H), dtype=torch.uint8, device=dev)
    xs = torch.empty((H // 128, M), dtype=torch.float32, device=dev)
    xr = torch.empty((M,), dtype=torch.float32, device=dev)
    y = torch.empty((M, H), dtype=torch.float32, device=dev)
    h = torch.empty((M, I), dtype=torch.float32, device=dev)
    lc.lacache_rmsnorm_f32(x, norm_w, y)
    lc.lacache_quant_rows_g(y, xq, xs, xr, lc.LACACHE_GRAN_TOKEN)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for i in range(reps):
            gq, gs, gr = sets["token"][i % S][:3]
            lc.lacache_gateup_swiglu_f32(xq, xs, gq, gs, gr, h)
    g.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(3):
        g.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    k_ms = e0.elapsed_time(e1) / (3 * reps)
    del g
    flop = 6.0 * M * H * I
    ach = 4.0 * M * H * I / (k_ms * 1e-3) / 1e12
    line = {
        "metric": "FP8 FFN TFLOP/s per layer at a quantization granularity (per token; per group and per tensor "
                  "beside it)",
        "value": round(flop / (ms["token"] * 1e-3) / 1e12, 3), "unit": "TFLOP/s", "n_gpus": 1, "steps": reps,
        "warmup": args.warmup, "ms_per_step": round(ms["token"], 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "fp8_e4m3 (fp32 accumulate)", "data": "synthetic",
        "config": {"workload": args.workload, "M": M, "H": H, "I": I, "granularity": "token", "weight_sets": S},
        "ms_per_step_by_granularity": {k: round(v, 5) for k, v in ms.items()},
        "tflops_by_granularity": {k: round(flop / (v * 1e-3) / 1e12, 1) for k, v in ms.items()},
        "error_vs_bf16_ffn": errs, "error_rows": rows,
        "timing": "HIP graph of %d back-to-back calls per granularity, 3 replays" % reps,
        "roofline": {"bound": "mfma", "achieved": round(ach, 1), "peak": PEAK_FP8_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(ach / PEAK_FP8_TFLOPS, 4), "traffic": None,
                     "kernel": "gateup_tiled (h-only, per-column scales)", "kernel_ms": round(k_ms, 5),
                     "algorithmic_flop": 4 * M * H * I},
    }
    print(json.dumps(line), flush=True)


def first_layer_main(args):
    """One line for the token-wise first layer (EmbedCache / RoPECache,
    Sec. 3.3) at the LLaDA-8B shape (H = 4096, 32 heads of 128, vocabulary
    126464): a step is the update of one 32-token block of a 512-token
    sequence (embedding + norm, QKV projection, RoPE + scatter of those rows);
    the full recompute of all 512 rows (the block's first step) is timed
    beside it. Inputs are seeded synthetic (token ids, embedding table,
    weights); 4 rotating QKV weight sets keep the projection streaming from
    HBM."""
    import numpy as np
    import torch

    import paper_2607_16339_amd as lc

    H, heads, N, vocab, Cn, D = 4096, 32, 512, 126464, 32, 128
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    lc.lib()
    g = torch.Generator(device="cpu").manual_seed(260716339)
    S = args.weight_sets

    def bf16_randn(shape, std):
        return (torch.randn(shape, generator=g) * std).to(torch.bfloat16).to(dev)

    embed = bf16_randn((vocab, H), 1.0)
    norm_w = (1.0 + torch.randn((H,), generator=g) * 0.02).to(torch.bfloat16).to(dev)
    wqkv = [bf16_randn((3 * heads * D, H), 0.02) for _ in range(S)]
    i = torch.arange(D // 2, dtype=torch.float64)
    ang = torch.arange(N, dtype=torch.float64)[:, None] * torch.pow(torch.tensor(500000.0, dtype=torch.float64),
                                                                     -2.0 * i / D)[None, :]
    rc, rs = torch.cos(ang).float().to(dev), torch.sin(ang).float().to(dev)
    caches = [torch.empty((N, H), dtype=torch.bfloat16, device=dev)] + [
        torch.empty((heads, N, D), dtype=torch.bfloat16, device=dev) for _ in range(3)]
    ids = torch.randint(0, vocab, (N,), generator=g, dtype=torch.int32).to(dev)
    rows_all = torch.arange(N, dtype=torch.int32, device=dev)
    c0 = N // 2 + Cn
    rows_c = torch.arange(c0, c0 + Cn, dtype=torch.int32, device=dev)
    ids_c = torch.randint(0, vocab, (Cn,), generator=g, dtype=torch.int32).to(dev)

    def call(t, rows, j):
        lc.lacache_first_layer_tokens(t, rows, embed, norm_w, wqkv[j % S], rc, rs, *caches)

    call(ids, rows_all, 0)
    stream = torch.cuda.current_stream()
    reps = max(min(args.steps, 64), 8)

    def timed(fn):
        for j in range(args.warmup):
            fn(j)
        torch.cuda.synchronize()
        gr = torch.cuda.CUDAGraph()
        with torch.cuda.graph(gr):
            for j in range(reps):
                fn(j)
        gr.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(3):
            gr.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        del gr
        return e0.elapsed_time(e1) / (3 * reps)

    ms_block = timed(lambda j: call(ids_c, rows_c, j))
    ms_full = timed(lambda j: call(ids, rows_all, j))
    # the dominant kernel of the block update: the QKV projection of 32 rows
    y = torch.empty((Cn, H), dtype=torch.bfloat16, device=dev)
    qkv = torch.empty((Cn, 3 * heads * D), dtype=torch.bfloat16, device=dev)
    ms_lin = timed(lambda j: lc.lacache_linear_bf16(y, wqkv[j % S], qkv))
    lin_bytes = 3 * heads * D * H * 2 + Cn * H * 2 + Cn * 3 * heads * D * 2
    gbs = lin_bytes / (ms_lin * 1e-3) / 1e9
    line = {
        "metric": "token-wise first layer (EmbedCache/RoPECache): 32-token block update, tokens/s",
        "value": round(Cn / (ms_block * 1e-3), 1), "unit": "tokens/s", "n_gpus": 1, "steps": reps,
        "warmup": args.warmup, "ms_per_step": round(ms_block, 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16 (fp32 accumulate)", "data": "synthetic",
        "config": {"workload": "first_layer_n512", "H": H, "heads": heads, "N": N, "block": Cn, "vocab": vocab,
                   "weight_sets": S},
        "ms_full_recompute_512_rows": round(ms_full, 5),
        "block_update_speedup_vs_full": round(ms_full / ms_block, 2),
        "timing": "HIP graph of %d back-to-back calls, 3 replays" % reps,
        "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                     "frac": round(gbs / PEAK_HBM_GBPS, 4), "traffic": None,
                     "kernel": "linear_bf16_kernel (QKV projection of the 32 block rows)",
                     "kernel_ms": round(ms_lin, 5), "algorithmic_bytes": lin_bytes},
    }
    if not args.no_cpu_baseline and not args.profile_only:
        import oracle.first_layer as F
        e = embed[ids_c.long()].view(torch.int16).cpu().numpy().view(np.uint16)
        wq = wqkv[0].view(torch.int16).cpu().numpy().view(np.uint16)
        nwh = norm_w.view(torch.int16).cpu().numpy().view(np.uint16)
        t0 = time.perf_counter()
        n = 0
        while time.perf_counter() - t0 < 10.0 and n < 16:
            _, yb = F.embed_norm(np.arange(Cn), e, nwh)
            F.linear_bf16(yb, wq)
            n += 1
        t = time.perf_counter() - t0
        line["cpu_baseline"] = {"value": round(n * Cn / t, 3), "unit": "tokens/s", "cores": _threads(),
                                "kind": "oracle",
                                "sample": "%d block updates of 32 rows (embedding + norm + QKV projection, fp64; "
                                          "RoPE excluded): %.2f s" % (n, t)}
    print(json.dumps(line), flush=True)


PEAK_BF16_TFLOPS = 2500.0  # dense bf16 MFMA


def attention_flop_bytes(w, mode):
    """Algorithmic FLOPs and HBM bytes of one FACache attention call. Plain
    and populate: every query row against every key (4 N^2 d per head: the
    score and the P V products). Resume: the rows of the 64-row query blocks
    inside U against the keys of the key blocks overlapping C only, the other
    rows against every key; their cached state (m, l, O~ in fp32) is read
    instead. Bytes: q, k, v read and o written once (bf16), plus the cache
    written (populate) or read (resume)."""
    N, d, B = w.N, w.d, 64
    cb0 = w.c_begin // B
    nc = (w.c_end + B - 1) // B - cb0 if w.c_begin < w.c_end else 0
    rows_u = N - nc * B
    if mode == 1:
        pairs = rows_u * nc * B + nc * B * N
    else:
        pairs = N * N
    flop = 4.0 * d * pairs * w.heads
    io = 4 * w.heads * N * d * 2
    cache = w.heads * rows_u * (2 + d) * 4 if mode in (0, 1) else 0
    return flop, io + cache


def attention_main(args):
    """One line for the first-layer FACache attention: a step is one resume
    call (a later denoising step of a SAR block, the FACache hot path); the
    plain and populate calls are timed beside it."""
    import numpy as np
    import torch

    import paper_2607_16339_amd as lc
    import synth

    w = synth.ATTN_WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    lc.lib()

    def dev_bf16(bits):
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16).copy()).view(torch.bfloat16).to(dev)

    q0, k0, v0 = (dev_bf16(a) for a in synth.make_qkv(w, step=0))
    q1, k1, v1 = (dev_bf16(a) for a in synth.make_qkv(w, step=1))
    o = torch.empty_like(q0)
    cm = torch.empty((w.heads, w.N), dtype=torch.float32, device=dev)
    cl = torch.empty_like(cm)
    co = torch.empty((w.heads, w.N, w.d), dtype=torch.float32, device=dev)

    def call(mode, q, k, v):
        lc.lacache_facache_attention(q, k, v, o, cache_m=cm, cache_l=cl, cache_o=co, c_begin=w.c_begin,
                                     c_end=w.c_end, mode=mode)

    # populate on step 0, then resume on step 1 (rows of C redrawn) must equal plain on step 1
    call(0, q0, k0, v0)
    call(1, q1, k1, v1)
    torch.cuda.synchronize()
    got = o.clone()
    call(2, q1, k1, v1)
    torch.cuda.synchronize()
    if not torch.equal(got.view(torch.int16), o.view(torch.int16)):
        raise RuntimeError("resume on a later step differs from plain attention of its inputs")

    stream = torch.cuda.current_stream()
    reps = max(min(args.steps, 64), 8)

    def time_mode(mode, q, k, v):
        for _ in range(args.warmup):
            call(mode, q, k, v)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(reps):
                call(mode, q, k, v)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        g.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        # untimed replays back to back for about WARM_S seconds, then the timed ones right behind them
        for _ in range(min(5000, int(WARM_S / max(e0.elapsed_time(e1) * 1e-3, 1e-6)) + 1)):
            g.replay()
        torch.cuda.synchronize()
        nrep = 3
        e0.record(stream)
        for _ in range(nrep):
            g.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        del g
        return e0.elapsed_time(e1) / (nrep * reps)

    ms = {"plain": time_mode(2, q1, k1, v1), "populate": time_mode(0, q0, k0, v0)}
    call(0, q0, k0, v0)  # the cache of step 0, then resume steps on step 1's inputs
    ms["resume"] = time_mode(1, q1, k1, v1)

    fl = {m: attention_flop_bytes(w, i)[0] for m, i in (("plain", 2), ("populate", 0), ("resume", 1))}
    by = {m: attention_flop_bytes(w, i)[1] for m, i in (("plain", 2), ("populate", 0), ("resume", 1))}
    tf = {m: fl[m] / (ms[m] * 1e-3) / 1e12 for m in ms}
    # the step's kernel is the resume call: about 40 FLOP per algorithmic byte,
    # far below the bf16 ridge (2500 / 8 = 312), so it is bound by HBM; the
    # plain call (2 N d FLOP per byte) is bound by the MFMA rate
    gbs = by["resume"] / (ms["resume"] * 1e-3) / 1e9
    roof = {"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
            "frac": round(gbs / PEAK_HBM_GBPS, 4), "traffic": None,
            "kernel": "facache_attention_kernel<1> (resume)", "kernel_ms": round(ms["resume"], 5),
            "algorithmic_bytes": by["resume"]}
    roof_plain = {"bound": "mfma", "achieved": round(tf["plain"], 1), "peak": PEAK_BF16_TFLOPS,
                  "unit": "TFLOP/s", "frac": round(tf["plain"] / PEAK_BF16_TFLOPS, 4),
                  "kernel": "facache_attention_kernel<2> (plain)", "kernel_ms": round(ms["plain"], 5),
                  "algorithmic_flop": fl["plain"]}
    line = {
        "metric": "FACache first-layer attention, resume step: tokens/s (bf16, d=128)",
        "value": round(w.heads * w.N / (ms["resume"] * 1e-3), 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": reps, "warmup": args.warmup, "ms_per_step": round(ms["resume"], 5), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16 (fp32 accumulate)", "data": "synthetic",
        "config": {"workload": w.name, "heads": w.heads, "N": w.N, "d": w.d, "c_begin": w.c_begin,
                   "c_end": w.c_end},
        "ms": {k: round(v, 5) for k, v in ms.items()},
        "tflops_algorithmic": {k: round(v, 1) for k, v in tf.items()},
        "hbm_GBps_algorithmic": {k: round(by[k] / (ms[k] * 1e-3) / 1e9, 1) for k in ms},
        "resume_speedup_vs_plain": round(ms["plain"] / ms["resume"], 3),
        "timing": "HIP graph of %d back-to-back calls per mode, 3 replays" % reps,
        "roofline": roof, "roofline_plain": roof_plain,
    }
    if not args.no_cpu_baseline and not args.profile_only:
        import oracle.attention as A
        bits = synth.make_qkv(w, step=1, heads=[0])
        t0 = time.perf_counter()
        n = 0
        while time.perf_counter() - t0 < 10.0 and n < 64:
            A.attention(*bits)
            n += 1
        t = time.perf_counter() - t0
        line["cpu_baseline"] = {"value": round(n * w.N / t, 3), "unit": "tokens/s", "cores": _threads(),
                                "kind": "oracle",
                                "sample": "%d plain attention calls of head 0 (%d x %d, fp64): %.2f s"
                                          % (n, w.N, w.d, t)}
    print(json.dumps(line), flush=True)


def _threads():
    try:
        from threadpoolctl import threadpool_info
        return max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # noqa: BLE001
        return os.cpu_count() or 1


if __name__ == "__main__":
    main()
