"""Throughput of the FoE per-cluster MoE block on one MI355X.

One step = one foe_cluster_block call (route -> permute -> grouped SwiGLU FFN
-> combine for every cluster, then the local reduction) on synthetic inputs
already resident in HBM.  Prints ONE JSON line.

  python bench.py [--gpus 1] [--steps K] [--warmup W] [--config NAME]
                  [--only] [--no-graph] [--cpu-seconds S]

Headline workload: the prefill-shaped cluster block with Zipf(1.2) router skew
(T=8192, d=2048, E=16, k=2, F=1024, bf16), where the expert FFN is bound by
the matrix cores.  The same line nests, under "workloads", one record per
other block workload -- decode (T=128, weight-streaming bound), large
(T=16384, d=4096, E=32, k=4, F=1536) and the 8-cluster layer share (C=8,
T=4096, E=8) -- each with its step time, tokens/s, expert-FFN TFLOP/s, the
roofline object of its dominant kernel and per-kernel fractions.  `--only`
(or any `--config`) measures the named workload alone.  Several independent
weight/input sets are rotated where one set is smaller than twice the
256 MB Infinity Cache.

`--config attn_share_bf16` (or another attention configuration) times the
per-group attention that feeds the block instead: one step = one
foe_group_attention call (H=8 groups, S=4096 tokens, d=2048, two query heads of
128 per group sharing its key/value head, causal).

`traffic` in the roofline object is the measured HBM traffic per launch of the
dominant kernel (rocprofv3 FETCH_SIZE + WRITE_SIZE, scaled by what the same
counters read for a plain copy of known size: `--copy-calibration`), read from
profiles/traffic.json; it is null when no measurement exists for this
workload or the kernel's source has changed since it was taken.

Timed passes per workload (both over K steps, HIP events on the library's
stream):
  A  plain steps, launched eagerly and (unless --no-graph) replayed from HIP
     graphs -> value / ms_per_step from the faster of the two (both times
     are reported; config.launch names the one used)
  B  the same steps with every kernel bracketed by HIP events (the library's
     timing hooks) -> per-kernel average duration and the roofline object
"""

from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "tokens/s and expert-FFN TFLOP/s per FoE cluster block (decode & prefill), 1 GPU"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
BF16_MFMA_PEAK_TFLOPS = 2500.0  # dense bf16 MFMA
FP32_VALU_PEAK_TFLOPS = 157.3   # fp32 vector
DEFAULT_CONFIG = "prefill_zipf_bf16"
# measured after the headline, in the same JSON line
NESTED_WORKLOADS = ("decode_bf16", "large_bf16", "layer_share_bf16")
MALL_BYTES = 256 << 20


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", default=None,
                    help=f"workload (default {DEFAULT_CONFIG} plus the nested block workloads)")
    ap.add_argument("--only", action="store_true",
                    help="measure the headline workload alone (no nested records)")
    ap.add_argument("--no-graph", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="budget of the oracle CPU baseline (0 = skip)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device copy 10 times (reference for "
                         "rocprofv3 FETCH_SIZE / WRITE_SIZE)")
    return ap.parse_args()


# kernel name (library timing hooks) -> source file that holds it
KERNEL_SOURCES = {"route": "route.hip", "permute_index": "permute.hip",
                  "permute_hist": "permute.hip", "permute_rank": "permute.hip",
                  "permute_scan": "permute.hip", "permute_scatter": "permute.hip",
                  "ffn_gateup": "ffn.hip", "ffn_down": "ffn.hip", "ffn_fused": "ffn.hip",
                  "ffn_gateup_f32": "ffn.hip",
                  "ffn_down_f32": "ffn.hip", "combine": "combine.hip", "reduce": "combine.hip",
                  "attn_qkv": "ffn.hip", "attn_out": "ffn.hip", "attn_prep": "attention.hip",
                  "attn_core": "attention.hip", "attn_xsum": "attention.hip"}


def source_sha(kernel):
    import hashlib
    src = KERNEL_SOURCES.get(kernel)
    if src is None:
        return None
    path = os.path.join(ROOT, "paper_2605_06206_amd", "csrc", src)
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def measured_traffic(config, kernel):
    """HBM bytes per launch measured with rocprofv3 counters for this workload
    and kernel, or None (no record, or the kernel source changed since)."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f).get(config, {}).get(kernel)
    if not rec or rec.get("source_sha256") != source_sha(kernel):
        return None
    return rec.get("bytes_per_launch")


def copy_calibration():
    import torch
    n = 1 << 30
    src = torch.ones(n // 2, dtype=torch.bfloat16, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(10):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "launches": 10}), flush=True)


def kernel_work(name, cfg, e_touched):
    """Algorithmic (flops, bytes) of ONE launch of kernel `name` in a
    foe_cluster_block step.  Every kernel runs once per step over all C
    clusters: routing, the index pass (absent when the decode FFN lists its
    experts' pairs itself), the two grouped FFN kernels (all C*E experts) and
    the combine + reduction.  `e_touched` = experts (over all clusters) that
    got rows."""
    if "nq" in cfg:
        return attention_work(name, cfg)
    T, d, E, k, F, C = cfg["T"], cfg["d"], cfg["E"], cfg["k"], cfg["F"], cfg["C"]
    s = 2 if cfg["dtype"] == "bf16" else 4
    R = T * k          # pairs per cluster
    CR = C * R         # permuted rows over all clusters
    if name == "route":
        # x once, every cluster's router matrix, (idx, w) per pair
        return 2.0 * C * T * d * E, T * d * s + C * E * d * s + 8.0 * CR
    if name in ("ffn_gateup", "ffn_gateup_f32"):
        return 4.0 * CR * d * F, 2.0 * e_touched * F * d * s + CR * d * s + CR * F * s
    if name in ("ffn_down", "ffn_down_f32"):
        return 2.0 * CR * F * d, 1.0 * e_touched * d * F * s + CR * F * s + CR * d * s
    if name == "ffn_fused":
        # both GEMMs in one launch: the three weight matrices of every touched
        # expert, the gathered x rows, h written and read back, y written
        return (6.0 * CR * d * F,
                3.0 * e_touched * F * d * s + CR * d * s + 2.0 * CR * F * s + CR * d * s)
    if name == "combine":
        # y rows of every cluster, their indices and weights, x, out
        return 2.0 * CR * d, CR * d * s + 8.0 * CR + 2.0 * T * d * s
    return 0.0, 0.0


def attention_work(name, cfg):
    """Algorithmic (flops, bytes) of ONE launch of kernel `name` in a
    foe_group_attention call (H groups, S tokens, nq query heads of dim hd per
    group, bf16).  The causal attention counts the scores and the value
    products of the S(S+1)/2 visible (query, key) pairs only."""
    H, S, d, nq, hd = cfg["H"], cfg["S"], cfg["d"], cfg["nq"], cfg["hd"]
    rows = H * S
    n_qkv = (nq + 2) * hd
    if name == "attn_qkv":
        return 2.0 * rows * d * n_qkv, 2.0 * (rows * d + H * n_qkv * d + rows * n_qkv)
    if name == "attn_prep":
        # q and k read and written back rotated; v read, written transposed
        # (keys padded to a multiple of 64)
        s_pad = -(-S // 64) * 64
        return 0.0, 2.0 * (2 * rows * (nq + 1) * hd + rows * hd + H * hd * s_pad)
    if name == "attn_core":
        # bytes: q, k and v once and o once (the query blocks' re-reads of k
        # and v are not algorithmic)
        return (4.0 * hd * nq * H * S * (S + 1) / 2,
                2.0 * (rows * n_qkv + rows * nq * hd))
    if name == "attn_xsum":
        # the H residual planes read once, their fp32 sum written once
        return 0.0, 2.0 * rows * d + 4.0 * S * d
    if name == "attn_out":
        # one product over the concatenated head outputs plus the residual
        # sum: o, w_o and the fp32 sum read once, r_full written once
        return (2.0 * rows * nq * hd * d,
                2.0 * (rows * nq * hd + H * d * nq * hd + S * d) + 4.0 * S * d)
    return 0.0, 0.0


def roofline(name, cfg, e_touched, avg_s):
    flops, nbytes = kernel_work(name, cfg, e_touched)
    if cfg["dtype"] == "f32" and name.startswith("ffn"):
        bound, peak, unit, achieved = "alu", FP32_VALU_PEAK_TFLOPS, "TFLOP/s", flops / avg_s / 1e12
    elif nbytes > 0 and flops / nbytes > BF16_MFMA_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9):
        bound, peak, unit, achieved = "mfma", BF16_MFMA_PEAK_TFLOPS, "TFLOP/s", flops / avg_s / 1e12
    else:
        bound, peak, unit, achieved = "hbm", HBM_PEAK_GBS, "GB/s", nbytes / avg_s / 1e9
    return {"kernel": name, "bound": bound, "achieved": round(achieved, 2), "peak": peak,
            "unit": unit, "frac": round(achieved / peak, 4), "traffic": None,
            "avg_us": round(avg_s * 1e6, 3), "flops_per_launch": flops,
            "bytes_per_launch": nbytes}


def cpu_threads():
    """(threads of the BLAS pools numpy uses, their names)."""
    import numpy  # noqa: F401  (loads the BLAS whose pools are listed)
    try:
        from threadpoolctl import threadpool_info
        pools = threadpool_info()
        threads = max([p.get("num_threads", 1) for p in pools] or [1])
        blas = ",".join(sorted({p.get("internal_api", "?") for p in pools}))
    except Exception:  # pragma: no cover - informational only
        threads, blas = os.cpu_count(), "unknown"
    return threads, blas


def cpu_baseline(cfg_name, budget_s):
    """The oracle as it stands, timed on this host's cores on a bounded sample."""
    import numpy as np

    import oracle
    from paper_2605_06206_amd import synth

    threads, blas = cpu_threads()
    cfg = dict(synth.CONFIGS[cfg_name])
    # a token prefix small enough for ~1 s per oracle call
    per_tok = cfg["C"] * (cfg["k"] * 6.0 * cfg["d"] * cfg["F"] + 2.0 * cfg["d"] * cfg["E"])
    T_s = int(max(16, min(cfg["T"], 2e9 / per_tok)))
    inp = synth.make_block_inputs(cfg_name, T=T_s) if T_s < cfg["T"] else synth.make_block_inputs(cfg_name)
    reps, t0 = 0, time.perf_counter()
    while True:
        oracle.cluster_block(inp["x"], inp["clusters"], cfg["k"])
        reps += 1
        el = time.perf_counter() - t0
        if el >= budget_s or reps >= 1000:
            break
    tok_s = reps * T_s / el
    return {"value": round(tok_s, 2), "unit": "tokens/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"{reps} oracle runs (fp64 numpy) of the block on the first {T_s} of "
                      f"{cfg['T']} tokens, {el:.1f} s, BLAS {blas}, "
                      f"affinity {len(os.sched_getaffinity(0))} cpus"}


def timed_on(stream, n_steps, run):
    """Milliseconds of n_steps calls of run(i), HIP events on `stream`."""
    import torch
    torch.cuda.synchronize()
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    a.record(stream)
    for i in range(n_steps):
        run(i)
    b.record(stream)
    torch.cuda.synchronize()
    return a.elapsed_time(b)


def kernel_profile(foe, n_steps, run):
    """Pass B: every library kernel bracketed by HIP events -> (total ms,
    {name: launches, avg_us, total_ms})."""
    foe.profile_reset()
    foe.profile_enable(True)
    t_b = run(n_steps)
    foe.profile_enable(False)
    kernels = {}
    for name in foe.profile_names():
        n, tot = foe.profile_kernel(name)
        kernels[name] = {"launches": n, "avg_us": round(tot / n * 1e3, 3), "total_ms": tot}
    foe.profile_reset()
    return t_b, kernels


def cpu_baseline_attention(cfg, inp, budget_s):
    """The attention oracle as it stands, on a bounded sample of query rows of
    every group (the keys and values up to the last sampled row are formed
    each time, as the definition needs)."""
    import numpy as np

    from oracle import attention_oracle as ao
    S = cfg["S"]
    rows = np.arange(0, S, max(1, S // 16))
    x = inp["x"].astype(np.float64)
    reps, t0 = 0, time.perf_counter()
    while True:
        for h, g in enumerate(inp["groups"]):
            ao.group_attention_rows(x[h], g["w_qkv"], g["w_o"], cfg["nq"], cfg["hd"],
                                    cfg["theta"], cfg["scale"], rows)
        reps += 1
        el = time.perf_counter() - t0
        if el >= budget_s or reps >= 100:
            break
    threads, blas = cpu_threads()
    return {"value": round(reps * len(rows) / el, 2), "unit": "tokens/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"{reps} oracle runs (fp64 numpy) of {len(rows)} query rows spread over "
                      f"the {S} positions, all {cfg['H']} groups, {el:.1f} s, BLAS {blas}"}


def main_attention(args):
    """One step = one foe_group_attention call (q/k/v projection, rotary
    embedding, causal attention, output projection, residual average over the
    groups) on one sequence resident in HBM."""
    import numpy as np
    import torch

    from paper_2605_06206_amd import foe, synth

    torch.cuda.set_device(0)
    dev = "cuda:0"
    inp = synth.make_attention_inputs(args.config)
    cfg = dict(inp["cfg"], name=args.config, dtype="bf16")
    H, S, d, nq, hd = cfg["H"], cfg["S"], cfg["d"], cfg["nq"], cfg["hd"]

    def up(a):
        return torch.from_numpy(synth.bf16_bits(a)).to(dev).view(torch.bfloat16)

    x = up(inp["x"])
    w_qkv = up(np.stack([g["w_qkv"] for g in inp["groups"]]))
    w_o = up(np.concatenate([g["w_o"] for g in inp["groups"]], axis=1))
    out = torch.empty((S, d), dtype=torch.bfloat16, device=dev)
    L = foe.lib()
    ws_n = L.foe_group_attention_workspace_bytes(H, S, d, nq, hd)
    ws = torch.empty(ws_n, dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()
    sraw = stream.cuda_stream
    call = (foe.BF16, H, S, d, nq, hd, float(cfg["theta"]), float(cfg["scale"]), x.data_ptr(),
            w_qkv.data_ptr(), w_o.data_ptr(), out.data_ptr(), ws.data_ptr(), ws_n)

    def step(i, s):
        rc = L.foe_group_attention(*call, s)
        if rc != 0:
            raise RuntimeError(foe.last_error())

    for i in range(args.warmup):
        step(i, sraw)
    eager_ms = timed_on(stream, args.steps, lambda i: step(i, sraw)) / args.steps
    graph_ms = None
    if not args.no_graph:
        side = torch.cuda.Stream()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=side):
            step(0, side.cuda_stream)
        step(0, sraw)
        torch.cuda.synchronize()
        ref = out.clone()
        out.zero_()
        g.replay()
        torch.cuda.synchronize()
        if not torch.equal(out, ref):
            raise RuntimeError("graph replay differs from the eager call")
        for _ in range(args.warmup):
            g.replay()
        graph_ms = timed_on(stream, args.steps, lambda i: g.replay()) / args.steps
    use_graph = graph_ms is not None and graph_ms < eager_ms
    ms = graph_ms if use_graph else eager_ms

    t_b, kernels = kernel_profile(
        foe, args.steps, lambda n: timed_on(stream, n, lambda i: step(i, sraw)))
    dom = max(kernels, key=lambda n: kernels[n]["total_ms"])
    roof = roofline(dom, cfg, 0, kernels[dom]["avg_us"] * 1e-6)
    roof["traffic"] = measured_traffic(args.config, dom)
    per_kernel_roof = {n: roofline(n, cfg, 0, v["avg_us"] * 1e-6)
                       for n, v in kernels.items() if sum(attention_work(n, cfg)) > 0}
    flops = sum(attention_work(n, cfg)[0] for n in ("attn_qkv", "attn_core", "attn_out"))
    line = {
        "metric": "tokens/s of the per-group attention feeding the FoE block, 1 GPU",
        "value": round(S / (ms * 1e-3), 2),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) activations, N(0,sigma) weights)",
        "config": {"workload": f"{args.config}: H={H} S={S} d={d} nq={nq} hd={hd} bf16, causal",
                   "H": H, "S": S, "d": d, "nq": nq, "hd": hd,
                   "launch": "hip_graph_replay" if use_graph else "eager"},
        "attention_tflops": round(flops / (ms * 1e-3) / 1e12, 3),
        "eager_ms_per_step": round(eager_ms, 6),
        "graph_ms_per_step": None if graph_ms is None else round(graph_ms, 6),
        "profiled_ms_per_step": round(t_b / args.steps, 6),
        "roofline": roof,
        "kernels": {n: {"avg_us": v["avg_us"], "launches_per_step": v["launches"] / args.steps,
                        **({"frac": per_kernel_roof[n]["frac"], "bound": per_kernel_roof[n]["bound"]}
                           if n in per_kernel_roof else {})}
                    for n, v in kernels.items()},
        "cpu_baseline": None,
    }
    if args.cpu_seconds > 0:
        line["cpu_baseline"] = cpu_baseline_attention(cfg, inp, args.cpu_seconds)
    print(json.dumps(line), flush=True)


def main():
    args = parse()
    if args.copy_calibration:
        copy_calibration()
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs on one GPU only: the library has no multi-GPU path "
              "(use --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2605_06206_amd import foe, synth

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    args.nested = args.config is None and not args.only
    if args.config is None:
        args.config = DEFAULT_CONFIG
    if args.config in synth.ATTN_CONFIGS:
        main_attention(args)
        return
    torch.cuda.set_device(0)
    # every workload's inputs are drawn and uploaded first (host work, GPU
    # idle); the timed passes then run back to back, the headline last
    names = (list(NESTED_WORKLOADS) if args.nested else []) + [args.config]
    measure = {name: prepare_block(args, name) for name in names}
    recs = {name: measure[name]() for name in names}
    line = recs[args.config]
    if args.nested:
        line["workloads"] = {}
        for name in NESTED_WORKLOADS:
            line["workloads"][name] = {key: recs[name][key] for key in (
                "value", "unit", "ms_per_step", "dtype", "config", "block_tflops",
                "expert_ffn_tflops", "eager_ms_per_step", "graph_ms_per_step",
                "profiled_ms_per_step", "roofline", "kernels")}
    if args.cpu_seconds > 0:
        line["cpu_baseline"] = cpu_baseline(args.config, args.cpu_seconds)
    print(json.dumps(line), flush=True)


def prepare_block(args, name):
    """Inputs of one block workload drawn and resident in HBM; returns the
    function that runs its passes A and B and returns its record (no CPU
    baseline)."""
    import numpy as np
    import torch

    from paper_2605_06206_amd import foe, synth

    dev = "cuda:0"
    cfg = dict(synth.CONFIGS[name], name=name)
    dt = cfg["dtype"]
    T, d, E, k, F, C = cfg["T"], cfg["d"], cfg["E"], cfg["k"], cfg["F"], cfg["C"]
    s_el = 2 if dt == "bf16" else 4
    set_bytes = C * (3 * E * F * d + E * d) * s_el + T * d * s_el
    nsets = int(min(8, max(1, math.ceil(2 * MALL_BYTES / set_bytes))))

    def up(a):
        if dt == "bf16":
            return torch.from_numpy(synth.bf16_bits(a)).to(dev).view(torch.bfloat16)
        return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(dev)

    sets = []
    for i in range(nsets):
        inp = synth.make_block_inputs(name, weight_set=i)
        cls = inp["clusters"]
        st = {"x": up(inp["x"])}
        for key in ("w_router", "w_gate", "w_up", "w_down"):
            st[key] = up(np.stack([c[key] for c in cls]))
        st["bias"] = (torch.from_numpy(np.stack([c["bias"] for c in cls])).to(dev)
                      if cls[0]["bias"] is not None else None)
        sets.append(st)
        del inp, cls

    L = foe.lib()
    dtc = foe.BF16 if dt == "bf16" else foe.F32
    ws_n = foe.workspace_bytes("cluster_block", dtc, C, T, d, E, k, F)
    ws = torch.empty(ws_n, dtype=torch.uint8, device=dev)
    out = torch.empty((T, d), dtype=sets[0]["x"].dtype, device=dev)
    scale = 1.0 / C
    stream = torch.cuda.current_stream()

    def ptr(t):
        return None if t is None else t.data_ptr()

    calls = [(dtc, C, T, d, E, k, F, ptr(st["x"]), ptr(st["w_router"]), ptr(st["bias"]),
              ptr(st["w_gate"]), ptr(st["w_up"]), ptr(st["w_down"]), scale, ptr(out), ptr(ws),
              ws_n) for st in sets]

    def step(i, s):
        rc = L.foe_cluster_block(*calls[i % nsets], s)
        if rc != 0:
            raise RuntimeError(foe.last_error())

    # experts (over all clusters) that received rows, for the weight-streaming
    # bytes; computed outside the timed region
    e_touched = 0
    for h in range(C):
        st = sets[0]
        idx, _ = foe.route(st["x"], st["w_router"][h], None if st["bias"] is None else st["bias"][h], k)
        p = foe.permute(idx, st["x"], E)
        e_touched += int((p["counts"] > 0).sum().item())

    def timed(n_steps, run):
        return timed_on(stream, n_steps, run)

    # the closure holds every buffer the raw pointers in `calls` point into
    # (inputs, workspace, output) until the workload has been measured
    keep = {"sets": sets, "ws": ws, "out": out}

    def run_measure():
        rec = measure_block(args, name, cfg, foe, stream, nsets, sets, calls, out, step, timed,
                            e_touched)
        keep.clear()
        return rec

    return run_measure


def measure_block(args, name, cfg, foe, stream, nsets, sets, calls, out, step, timed, e_touched):
    """Passes A and B of one prepared block workload; returns its record."""
    import torch

    dt = cfg["dtype"]
    T, d, E, k, F, C = cfg["T"], cfg["d"], cfg["E"], cfg["k"], cfg["F"], cfg["C"]
    sraw = stream.cuda_stream
    for i in range(args.warmup):
        step(i, sraw)
    eager_ms = timed(args.steps, lambda i: step(i, sraw)) / args.steps

    graph_ms = None
    if not args.no_graph:
        graphs = []
        side = torch.cuda.Stream()
        for i in range(nsets):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=side):
                step(i, side.cuda_stream)
            graphs.append(g)
        # a replay must reproduce the eager result bit for bit
        step(0, sraw)
        torch.cuda.synchronize()
        ref = out.clone()
        out.zero_()
        graphs[0].replay()
        torch.cuda.synchronize()
        if not torch.equal(out, ref):
            raise RuntimeError("graph replay differs from the eager block")
        for i in range(args.warmup):
            graphs[i % nsets].replay()
        graph_ms = timed(args.steps, lambda i: graphs[i % nsets].replay()) / args.steps
    # both launch modes time the same steps; the faster one is the throughput
    use_graph = graph_ms is not None and graph_ms < eager_ms
    ms = graph_ms if use_graph else eager_ms

    # pass B: per-kernel HIP events (eager launches on the same stream)
    t_b, kernels = kernel_profile(foe, args.steps, lambda n: timed(n, lambda i: step(i, sraw)))
    dom = max(kernels, key=lambda n: kernels[n]["total_ms"])
    roof = roofline(dom, cfg, e_touched, kernels[dom]["avg_us"] * 1e-6)
    roof["traffic"] = measured_traffic(name, dom)
    per_kernel_roof = {n: roofline(n, cfg, e_touched, v["avg_us"] * 1e-6)
                       for n, v in kernels.items() if kernel_work(n, cfg, e_touched)[1] > 0}

    ffn_ms = sum(v["total_ms"] for n, v in kernels.items() if n.startswith("ffn")) / args.steps
    tokens_s = T / (ms * 1e-3)
    flops = C * (2.0 * T * d * E + 6.0 * T * k * d * F)
    line = {
        "metric": METRIC,
        "value": round(tokens_s, 2),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": dt,
        "data": "synthetic (seeded N(0,1) activations, N(0,sigma) weights; "
                f"{nsets} rotated input/weight sets)",
        "config": {"workload": f"{name}: C={C} T={T} d={d} E={E} k={k} F={F} {dt}",
                   "C": C, "T": T, "d": d, "E": E, "k": k, "F": F,
                   "launch": "hip_graph_replay" if use_graph else "eager"},
        "block_tflops": round(flops / (ms * 1e-3) / 1e12, 3),
        "expert_ffn_tflops": round(6.0 * C * T * k * d * F / (ffn_ms * 1e-3) / 1e12, 3),
        "eager_ms_per_step": round(eager_ms, 6),
        "graph_ms_per_step": None if graph_ms is None else round(graph_ms, 6),
        "profiled_ms_per_step": round(t_b / args.steps, 6),
        "roofline": roof,
        "kernels": {n: {"avg_us": v["avg_us"], "launches_per_step": v["launches"] / args.steps,
                        **({"frac": per_kernel_roof[n]["frac"], "bound": per_kernel_roof[n]["bound"]}
                           if n in per_kernel_roof else {})}
                    for n, v in kernels.items()},
        "cpu_baseline": None,
    }
    sets.clear()
    calls.clear()
    return line




if __name__ == "__main__":
    main()
