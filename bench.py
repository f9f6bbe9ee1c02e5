#!/usr/bin/env python3
"""Benchmark of the chunked causal attention hot path on one MI355X.

A step is one forward walk over all chunks (each chunk's Q/K/V/O/LSE
offloaded to pinned host memory after its forward, except the last chunk)
followed by the reverse backward walk (offloaded chunks prefetched two
chunks ahead), on synthetic N(0,1) bf16 inputs already resident in HBM.

Reported (one JSON line):
  value          algorithmic TFLOP/s of the step with offload on; the
                 algorithmic count is 14*B*Hq*D per visible (query, key)
                 pair (forward QK^T, PV; backward the five products), the
                 causal half only
  pct_peak       value / 2516.6 TFLOP/s (256 CU x 2.4 GHz x 4096 bf16
                 flop/clk/CU, dense)
  offload_hidden 1 - max(0, T_on - T_off) / T_copy, where T_on and T_off are
                 the step with and without offload, timed in alternating
                 steps (so drift over the run falls on both), and T_copy the
                 event-timed copy busy time per step; the same for the
                 Q/O/LSE-only walk (offload.round_trip_qol) and the
                 K/V-evicting walk (offload.evict)
  ms_per_step_median / _min   over the K headline steps (an event between
                 steps)
  offload.per_chunk_exposed_ms   per forward / backward chunk, duration with
                 offload minus without (one marked step of each)
  offload_policy equal vs FLOPs-balanced chunk boundaries, each with the full
                 offload set and with the sequence-aware plan (row prefix per
                 chunk sized so its copy fits under the next chunk's forward
                 at the isolated link rate): step time, hidden fraction,
                 bytes, and the modelled peak of offloadable activations
  offload.link   the library's copy path alone (sppo_link_probe, 1 GiB):
                 GB/s device->host, host->device and both at once; with it
                 copy_iso_ms_per_step and hidden_pct_vs_iso
  roofline       the dominant kernel (largest summed time), from HIP events
                 around every launch on the compute stream in K further timed
                 steps (kept out of the headline steps)
  --sweep-n      replaces all of the above by one line per chunk count
  cpu_baseline   the fp64 oracle on a bounded sample (two heads, a prefix of
                 the sequence), in algorithmic TFLOP/s, with the CPU model and
                 extrapolated_full_step_s: the whole step's algorithmic flop at
                 that rate (an extrapolation, not a measurement)
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
PEAK_BF16_TFLOPS = 256 * 2.4e9 * 4096 / 1e12  # dense bf16 MFMA, MI355X
HBM_PEAK_GBS = 8000.0
METRIC = "chunked causal attn fwd+bwd TFLOP/s (% bf16 MFMA peak) + % offload hidden"

WORKLOADS = {
    # name: (S, N, Hq, Hkv, D, offload)
    "s128k_n16_offload": (131072, 16, 32, 32, 128, "qkvol"),
    "s32k_n8": (32768, 8, 32, 32, 128, "none"),
    "s512k_n32_gqa_offload": (524288, 32, 32, 8, 128, "qkvol"),
    "s1m_n64_offload": (1048576, 64, 32, 32, 128, "qkvol"),
}
DEFAULT_WORKLOAD = "s128k_n16_offload"


def pairs_per_chunk(offsets):
    """Visible (query, key) pairs of each chunk: s_i * c_i + s_i (s_i + 1) / 2."""
    out = []
    for i in range(len(offsets) - 1):
        c, s = offsets[i], offsets[i + 1] - offsets[i]
        out.append(s * c + s * (s + 1) // 2)
    return out


def algorithmic_flops(offsets, B, Hq, D):
    """Per kernel, summed over chunks: fwd 4D, dkdv 8D (S, dP, dV, dK), dq 2D
    (dQ; its S/dP recomputation is not credited) per visible pair and head."""
    p = sum(pairs_per_chunk(offsets)) * B * Hq * D
    return {"fwd": 4 * p, "bwd_dkdv": 8 * p, "bwd_dq": 2 * p, "bwd_pre": 0, "total": 14 * p}


def cpu_model():
    """The host CPU as /proc/cpuinfo names it: model name, family, model and
    stepping, and the number of logical CPUs it lists."""
    fields, n = {}, 0
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                key, _, val = line.partition(":")
                key = key.strip()
                if key == "processor":
                    n += 1
                if key in ("model name", "cpu family", "model", "stepping", "vendor_id") and key not in fields:
                    fields[key] = val.strip()
    except OSError:
        return "unknown"
    return (f"{fields.get('model name', 'unknown')} ({fields.get('vendor_id', '?')}, family "
            f"{fields.get('cpu family', '?')} model {fields.get('model', '?')} stepping "
            f"{fields.get('stepping', '?')}; {n} logical CPUs listed)")


def cpu_threads():
    """Host threads for the oracle: the CPUs this process may run on, capped
    by the OpenMP thread limit of the environment (the CPU share of one GPU
    on a shared box), and the affinity count itself."""
    affinity = len(os.sched_getaffinity(0))
    cap = os.environ.get("OMP_NUM_THREADS", "")
    n = min(affinity, int(cap)) if cap.isdigit() and int(cap) > 0 else affinity
    return n, affinity


def oracle_cpu_baseline(inp, D, sample_tokens, sample_heads):
    """Time the fp64 oracle (fwd + bwd, unchunked) on the first
    ``sample_heads`` heads over the first ``sample_tokens`` tokens of the same
    inputs (heads one after another, as the oracle runs them)."""
    import numpy as np

    import oracle

    def host(t):
        return t[:, :sample_tokens, :sample_heads].float().cpu().numpy().astype(np.float64)

    from threadpoolctl import threadpool_limits

    q, k, v, do = host(inp["q"]), host(inp["k"]), host(inp["v"]), host(inp["do"])
    cores, affinity = cpu_threads()
    with threadpool_limits(cores):
        t0 = time.perf_counter()
        oracle.attention(q, k, v, do, 1.0 / math.sqrt(D))
        dt = time.perf_counter() - t0
    flops = 14 * D * sample_heads * sample_tokens * (sample_tokens + 1) / 2
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": int(cores), "kind": "oracle",
            "affinity_cpus": affinity,
            "sample": f"fp64 NumPy oracle, unchunked fwd+bwd of heads 0..{sample_heads - 1} over the "
                      f"first {sample_tokens} tokens ({flops:.3e} algorithmic flop in {dt:.2f} s)",
            "seconds": dt}


def kernel_source_hash(kernel):
    """sha256 of the HIP source that defines ``kernel``."""
    import hashlib

    src = {"fwd": "attn_fwd_bf16.hip", "bwd_dkdv": "attn_bwd_bf16.hip", "bwd_dq": "attn_bwd_bf16.hip",
           "bwd_pre": "attn_bwd_bf16.hip"}[kernel]
    path = os.path.join(ROOT, "paper_2503_10377_amd", "csrc", src)
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def measured_traffic(kernel, workload):
    """HBM bytes per launch of ``kernel`` from the committed counter record
    (profiles/<kernel>_<workload>_traffic.json), or None when the record is
    missing or the kernel source changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("source_sha256") != kernel_source_hash(kernel):
        return None
    return rec.get("bytes_per_launch")


def walk_memory(run_step, walk):
    """Device memory a chunk walk needs (see device_memory in main)."""
    import gc

    import torch

    torch.cuda.synchronize()
    walk.arena = walk.keep = walk._layout = None
    gc.collect()  # nothing else is freed inside the measured step
    base = torch.cuda.memory_allocated()
    torch.cuda.reset_peak_memory_stats()
    run_step()
    torch.cuda.synchronize()
    return {"walk_peak_GiB": (torch.cuda.max_memory_allocated() - base) / 2**30,
            "saved_activation_GiB": (walk.arena.nbytes + walk.keep.nbytes) / 2**30,
            "arena_GiB": walk.arena.nbytes / 2**30, "keep_GiB": walk.keep.nbytes / 2**30,
            "arena_high_water_GiB": walk.arena.high_water / 2**30}


def copy_calibration(nbytes):
    """A plain device-to-device copy of ``nbytes``, three times: the known
    traffic against which FETCH_SIZE / WRITE_SIZE are scaled."""
    import torch

    src = torch.ones(nbytes, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": nbytes, "copies": 3}), flush=True)


def sweep_chunk_count(args, inp, S, Hq, Hkv, D, counts):
    """Chunk-count trade-off on one GPU: for each N, the forward walk alone
    and the full forward + backward walk (no offload), timed with events
    over args.steps steps after args.warmup."""
    import torch

    from paper_2503_10377_amd.chunked import ChunkedAttention

    st = torch.cuda.current_stream()
    for n in counts:
        ca = ChunkedAttention(1, S, n, Hq, Hkv, D, dtype="bf16", offload="none")
        out = ca.alloc_outputs()
        fl = algorithmic_flops(ca.offsets, 1, Hq, D)
        row = {"sweep": "chunk_count", "seq_len": S, "n_chunks": n, "chunk_len": S // n, "n_q_heads": Hq,
               "n_kv_heads": Hkv, "head_dim": D, "steps": args.steps}
        for phase, run in (("fwd", lambda: ca.forward_only(inp, out)),
                           ("fwd_bwd", lambda: ca.step(inp, out, export=False))):
            for _ in range(args.warmup):
                run()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(st)
            for _ in range(args.steps):
                run()
            e1.record(st)
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / args.steps
            f = fl["fwd"] if phase == "fwd" else fl["total"]
            row[f"{phase}_ms"] = ms
            row[f"{phase}_tflops"] = f / (ms * 1e-3) / 1e12
            row[f"{phase}_pct_peak"] = 100.0 * row[f"{phase}_tflops"] / PEAK_BF16_TFLOPS
        ca.close()
        print(json.dumps(row), flush=True)


LAYER_WORKLOAD = (131072, 16, 32, 32, 128)  # S, N, Hq, Hkv, D (width 4096, MLP 16384)
LAYER_METRIC = "full-layer chunked fwd+bwd TFLOP/s (% bf16 MFMA peak) + % offload hidden"


def layer_cpu_baseline(inp, p, Hq, Hkv, D, sample_tokens):
    """Time the fp64 layer oracle (fwd + bwd, unchunked) over the first
    ``sample_tokens`` tokens of the same inputs and weights."""
    import numpy as np

    from oracle import transformer_layer as T

    host = lambda t: t.float().cpu().numpy().astype(np.float64)
    x, dy = host(inp["x"][:sample_tokens]), host(inp["dy"][:sample_tokens])
    hp = {k: host(v) for k, v in p.items()}
    from threadpoolctl import threadpool_limits

    from paper_2503_10377_amd.chunked_layer import ChunkedLayer
    cores, affinity = cpu_threads()
    flops, _ = ChunkedLayer.flops(sample_tokens, [0, sample_tokens], Hq, Hkv, D)
    with threadpool_limits(cores):
        t0 = time.perf_counter()
        T.layer(x, dy, hp, Hq, Hkv, D)
        dt = time.perf_counter() - t0
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": int(cores), "kind": "oracle",
            "affinity_cpus": affinity,
            "sample": f"fp64 NumPy layer oracle, unchunked fwd+bwd of the full layer over the first "
                      f"{sample_tokens} tokens ({flops:.3e} algorithmic flop in {dt:.2f} s)"}


def layer_bench(args):
    """One JSON line for the full-layer chunk walk (LayerNorm, QKV / output
    projections, chunked causal attention, MLP) on the 128K-token workload.
    The walk with the non-K/V activations offloaded and the same walk
    without offload are timed in alternating steps (so clock drift over the
    run falls on both alike); per-op-class times come from events around
    every library call in one further step of each."""
    import torch

    from paper_2503_10377_amd import sppo as L
    from paper_2503_10377_amd.chunked_layer import ChunkedLayer
    from paper_2503_10377_amd.inputs import make_layer_inputs

    S, N, Hq, Hkv, D = LAYER_WORKLOAD
    torch.cuda.init()
    inp, p = make_layer_inputs(S, Hq, Hkv, D, seed=0, device="cuda")
    st = torch.cuda.current_stream()
    offload = args.layer_offload
    print(f"[bench] layer S={S} N={N} Hq={Hq} Hkv={Hkv} D={D} offload={offload}", file=sys.stderr, flush=True)
    lay = ChunkedLayer(S, N, Hq, Hkv, D, offload=offload)
    has_copy = lay.offload != L.SPPO_OFFLOAD_NONE
    lay_off = ChunkedLayer(S, N, Hq, Hkv, D, offload="none") if has_copy and not args.no_offload_compare else None
    walks = [lay] + ([lay_off] if lay_off else [])
    out = lay.alloc_outputs()
    for _ in range(args.warmup):
        for w in walks:
            w.step(inp, p, out, lookahead=args.lookahead)
    torch.cuda.synchronize()
    if has_copy:
        L.sppo_copy_stats(lay.ctx, reset_after=True)
    times = [[] for _ in walks]
    for n in range(args.steps):
        for w, t in zip(walks, times):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(st)
            w.step(inp, p, out, lookahead=args.lookahead)
            e1.record(st)
            t.append((e0, e1))
    torch.cuda.synchronize()
    times = [[e0.elapsed_time(e1) for e0, e1 in t] for t in times]
    cs = L.sppo_copy_stats(lay.ctx, reset_after=True) if has_copy else None

    def breakdown(w):
        ops, marks = [], []
        w.step(inp, p, out, lookahead=args.lookahead, ops=ops, marks=marks)
        torch.cuda.synchronize()
        cats = {}
        for cat, flop, e0, e1 in ops:
            c = cats.setdefault(cat, {"ms": 0.0, "launches": 0, "flop": 0})
            c["ms"] += e0.elapsed_time(e1)
            c["launches"] += 1
            c["flop"] += flop
        span = {marks[n][0]: marks[n][1].elapsed_time(marks[n + 1][1]) for n in range(len(marks) - 1)}
        return cats, {"fwd_ms": sum(span[("fwd", i)] for i in range(w.N)),
                      "bwd_ms": sum(span[("bwd", i)] for i in range(w.N))}

    cats, ph_on = breakdown(lay)
    total, gemm_flop = ChunkedLayer.flops(S, lay.offsets, Hq, Hkv, D)
    per_on = sorted(times[0])
    ms_on = sum(per_on) / len(per_on)
    tflops = total / (ms_on * 1e-3) / 1e12
    res = {"metric": LAYER_METRIC, "value": tflops, "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "ms_per_step": ms_on, "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
           "pct_peak": 100.0 * tflops / PEAK_BF16_TFLOPS,
           "ms_per_step_median": per_on[len(per_on) // 2], "ms_per_step_min": per_on[0],
           "ms_steps": [round(t, 2) for t in times[0]],
           "tokens_per_s": S / (ms_on * 1e-3),
           "flop_per_step": {"total": total, "gemm": gemm_flop, "attention": total - gemm_flop},
           "config": {"workload": f"one pre-LayerNorm transformer layer fwd+bwd (width {Hq * D}, MLP {4 * Hq * D}, "
                                  f"{Hq} query / {Hkv} KV heads x head_dim {D}), batch 1, seq {S} in {N} chunks "
                                  f"of {S // N}, bf16 in / fp32 accumulate, offload {offload} (all chunks but "
                                  f"the last), prefetch lookahead {args.lookahead}",
                      "name": f"layer_s{S // 1024}k_n{N}", "seq_len": S, "n_chunks": N, "n_q_heads": Hq,
                      "n_kv_heads": Hkv, "head_dim": D, "hidden": Hq * D, "offload": offload}}
    kern = {}
    for cat, c in sorted(cats.items()):
        k = {"ms_per_step": c["ms"], "launches_per_step": c["launches"]}
        if c["flop"]:
            k["tflops"] = c["flop"] / (c["ms"] * 1e-3) / 1e12
        kern[cat] = k
    g = [c for cat, c in cats.items() if cat.startswith("gemm")]
    gms, gfl = sum(c["ms"] for c in g), sum(c["flop"] for c in g)
    kern["gemm_all"] = {"ms_per_step": gms, "launches_per_step": sum(c["launches"] for c in g),
                        "tflops": gfl / (gms * 1e-3) / 1e12}
    res["kernels"] = kern
    res["phases_ms"] = ph_on
    dom = max((n for n in kern if n != "gemm_all" and "tflops" in kern[n]), key=lambda n: kern[n]["ms_per_step"])
    ach = kern[dom]["tflops"]
    res["roofline"] = {"kernel": dom, "bound": "mfma", "achieved": ach, "peak": PEAK_BF16_TFLOPS,
                       "unit": "TFLOP/s", "frac": ach / PEAK_BF16_TFLOPS, "traffic": None}
    if cs is not None:
        steps = args.steps
        copy_ms = (cs["ms_d2h"] + cs["ms_h2d"]) / steps
        off = {"bytes_per_row": lay.offload_bytes_per_row(),
               "bytes_d2h_per_step": cs["bytes_d2h"] / steps, "bytes_h2d_per_step": cs["bytes_h2d"] / steps,
               "copy_ms_per_step": copy_ms,
               "d2h_GBps": cs["bytes_d2h"] / max(cs["ms_d2h"], 1e-9) / 1e6,
               "h2d_GBps": cs["bytes_h2d"] / max(cs["ms_h2d"], 1e-9) / 1e6}
        if lay_off is not None:
            mem_on = walk_memory(lambda: lay.step(inp, p, out, lookahead=args.lookahead), lay)
            mem_off = walk_memory(lambda: lay_off.step(inp, p, out, lookahead=args.lookahead), lay_off)
            off["device_memory"] = {"offload": mem_on, "no_offload": mem_off,
                                    "saved_GiB": mem_off["walk_peak_GiB"] - mem_on["walk_peak_GiB"]}
            per_off = sorted(times[1])
            ms_off = sum(per_off) / len(per_off)
            _, ph_off = breakdown(lay_off)
            exposed = max(0.0, ms_on - ms_off)
            off["ms_per_step_no_offload"] = ms_off
            off["ms_steps_no_offload"] = [round(t, 2) for t in times[1]]
            off["phases_ms_no_offload"] = ph_off
            off["exposed_ms_per_step"] = exposed
            off["hidden_pct"] = 100.0 * max(0.0, min(1.0, 1.0 - exposed / copy_ms)) if copy_ms > 0 else None
        res["offload"] = off
        res["offload_hidden_pct"] = off.get("hidden_pct")
    for w in walks:
        w.close()
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU layer oracle sample", file=sys.stderr, flush=True)
        res["cpu_baseline"] = layer_cpu_baseline(inp, p, Hq, Hkv, D, args.layer_cpu_tokens)
        res["cpu_baseline"]["cpu_model"] = cpu_model()
        # an extrapolation from the measured rate, not a measurement
        res["cpu_baseline"]["extrapolated_full_step_s"] = total / (res["cpu_baseline"]["value"] * 1e12)
    print(json.dumps(res), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD, choices=sorted(WORKLOADS))
    ap.add_argument("--lookahead", type=int, default=2)
    ap.add_argument("--cpu-sample-tokens", type=int, default=32768)
    ap.add_argument("--cpu-sample-heads", type=int, default=2)
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="only run a device copy of BYTES (counter calibration) and exit")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-offload-compare", action="store_true")
    ap.add_argument("--no-policy", action="store_true", help="skip the partition / offload-ratio comparison")
    ap.add_argument("--sweep-n", default="", metavar="N1,N2,...",
                    help="instead of the headline line: one JSON line per chunk count N at the workload's S and "
                         "heads, no offload (forward and forward+backward time and %% of peak)")
    ap.add_argument("--layer", action="store_true",
                    help="instead of the headline line: the full-layer chunk walk (projections, attention, MLP) "
                         "at seq 131072 in 16 chunks, width 4096")
    ap.add_argument("--layer-offload", default="qol", choices=("none", "qol", "qkvol", "qkvol_evict"))
    ap.add_argument("--layer-cpu-tokens", type=int, default=4096)
    args = ap.parse_args()
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the sharded path is "
              "described, not built.", file=sys.stderr)
        sys.exit(2)

    if args.layer:
        layer_bench(args)
        return

    import torch

    from paper_2503_10377_amd import sppo as L
    from paper_2503_10377_amd.chunked import ChunkedAttention
    from paper_2503_10377_amd.inputs import make_inputs

    S, N, Hq, Hkv, D, offload = WORKLOADS[args.workload]
    B = 1
    torch.cuda.init()
    inp = make_inputs(B, S, Hq, Hkv, D, torch.bfloat16, seed=0, device="cuda")
    if args.sweep_n:
        sweep_chunk_count(args, inp, S, Hq, Hkv, D, [int(x) for x in args.sweep_n.split(",")])
        return
    ca = ChunkedAttention(B, S, N, Hq, Hkv, D, dtype="bf16", offload=offload)
    out = ca.alloc_outputs(export=False)
    flops = algorithmic_flops(ca.offsets, B, Hq, D)

    def timed(c, steps, timing, o=None):
        o = out if o is None else o
        for _ in range(args.warmup):
            c.step(inp, o, lookahead=args.lookahead)
        torch.cuda.synchronize()
        print(f"[bench] warmup done (offload {c.offload}, kernel events {bool(timing)})", file=sys.stderr, flush=True)
        L.sppo_copy_stats(c.ctx, reset_after=True)
        L.sppo_set_kernel_timing(c.ctx, timing)
        L.sppo_kernel_times(c.ctx, reset_after=True)
        st = torch.cuda.current_stream()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
        torch.cuda.synchronize()
        ev[0].record(st)
        for n in range(steps):
            c.step(inp, o, lookahead=args.lookahead)
            ev[n + 1].record(st)
        torch.cuda.synchronize()
        ms = ev[0].elapsed_time(ev[steps]) / steps
        step_times.append([ev[n].elapsed_time(ev[n + 1]) for n in range(steps)])
        kt = L.sppo_kernel_times(c.ctx, reset_after=True)
        cs = L.sppo_copy_stats(c.ctx, reset_after=True) if c.offload != L.SPPO_OFFLOAD_NONE else None
        L.sppo_set_kernel_timing(c.ctx, False)
        return ms, kt, cs

    step_times = []

    def alternate(walks, steps, o=None):
        """Time several walks in alternating steps: args.warmup steps of each,
        then `steps` rounds of one event-timed step of each in turn.
        Returns per walk the mean ms per step, the step times and the copy
        statistics of the timed steps (None without offload)."""
        o = out if o is None else o
        for w in walks.values():
            for _ in range(args.warmup):
                w.step(inp, o, lookahead=args.lookahead)
        torch.cuda.synchronize()
        for w in walks.values():
            if w.offload != L.SPPO_OFFLOAD_NONE:
                L.sppo_copy_stats(w.ctx, reset_after=True)
        st = torch.cuda.current_stream()
        ev = {k: [] for k in walks}
        for n in range(steps):
            for k, w in walks.items():
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(st)
                w.step(inp, o, lookahead=args.lookahead)
                e1.record(st)
                ev[k].append((e0, e1))
            torch.cuda.synchronize()
            print(f"[bench] alternating round {n + 1}/{steps} ({', '.join(walks)})", file=sys.stderr, flush=True)
        res_ = {}
        for k, w in walks.items():
            t = [e0.elapsed_time(e1) for e0, e1 in ev[k]]
            cs_ = L.sppo_copy_stats(w.ctx, reset_after=True) if w.offload != L.SPPO_OFFLOAD_NONE else None
            res_[k] = {"ms": sum(t) / len(t), "steps": t, "cs": cs_}
        return res_

    def chunk_fwd_ms(c, o):
        """Forward duration of each chunk, from one step with an event at
        every chunk boundary."""
        marks = []
        c.step(inp, o, lookahead=args.lookahead, marks=marks)
        torch.cuda.synchronize()
        span = {marks[n][0]: marks[n][1].elapsed_time(marks[n + 1][1]) for n in range(len(marks) - 1)}
        return [span[("fwd", i)] for i in range(c.N)]

    def device_memory(c, o):
        """Measured device memory of one walk: its buffers for the chunks'
        saved activations are dropped, so the walk plans and allocates them
        again inside one measured step; torch's peak of allocated bytes over
        that step minus what was allocated before it is the walk's own
        device memory (arena, keep buffers and anything else a step
        allocates), independent of other walks alive in the process."""
        return walk_memory(lambda: c.step(inp, o, lookahead=args.lookahead), c)

    def modelled_peak_bytes(t_fwd, lens, rows, copy_row, freed_row, bw_GBps):
        """Peak device bytes of the chunks' offloadable activations (Q, O,
        LSE) during the forward walk, when each offloaded prefix is freed as
        soon as its copy lands: copies leave in chunk order (one FIFO
        stream), copy i starts at max(end of fwd i, end of copy i-1) and
        takes rows_i * copy_row / bw; chunk i's set is live from the start
        of fwd i.  Measured forward times and link rate, modelled frees."""
        bw = bw_GBps * 1e6  # bytes per ms
        start = [0.0]
        for t in t_fwd:
            start.append(start[-1] + t)
        end, prev = [], 0.0
        for i, r in enumerate(rows):
            begin = max(start[i + 1], prev)
            prev = begin + r * copy_row / bw
            end.append(prev)
        peak = 0.0
        for i in range(len(lens)):
            live = sum(lens[j] * freed_row for j in range(i + 1))
            freed = sum(rows[j] * freed_row for j in range(i) if end[j] <= start[i])
            peak = max(peak, live - freed)
        return peak

    def policy_compare(bw_GBps):
        """Sequence-aware offloading (NEXT-1): equal vs FLOPs-balanced chunk
        boundaries, each with the full offload set and with the planned row
        prefix per chunk (copy of chunk i bounded by the forward of chunk
        i+1 at the isolated link rate); the walks without offload, with the
        full set and with the plan are timed in alternating steps."""
        result = {}
        freed_row = B * (2 * Hq * D * 2 + 4 * Hq)
        for part in ("equal", "balanced"):
            offs = None if part == "equal" else L.sppo_balanced_offsets(S, N, 128)
            c_none = ChunkedAttention(B, S, N, Hq, Hkv, D, dtype="bf16", offsets=offs, offload="none")
            o = c_none.alloc_outputs(export=False)
            c_none.step(inp, o, lookahead=args.lookahead)
            t_fwd = chunk_fwd_ms(c_none, o)
            lens = [c_none.chunk_len(i) for i in range(N)]
            walks = {"none": c_none}
            for name in ("full", "plan"):
                walks[name] = ChunkedAttention(B, S, N, Hq, Hkv, D, dtype="bf16", offsets=offs, offload="qkvol")
            copy_row = walks["full"].offload_bytes_per_row()
            rows_of = {"full": lens[:-1] + [0],
                       "plan": L.sppo_plan_offload_rows(c_none.offsets, copy_row, bw_GBps, t_fwd[1:] + [0.0], 128)}
            for name in ("full", "plan"):
                walks[name].set_offload_rows(rows_of[name])
            alt = alternate(walks, steps, o)  # steps of the three walks in turn
            ms_none = alt["none"]["ms"]
            entry = {"offsets": c_none.offsets, "ms_per_step_no_offload": ms_none,
                     "ms_steps_no_offload": [round(x, 2) for x in alt["none"]["steps"]], "fwd_ms_per_chunk": t_fwd,
                     "device_memory_no_offload": device_memory(c_none, o)}
            for name in ("full", "plan"):
                rows, ms, cs_p = rows_of[name], alt[name]["ms"], alt[name]["cs"]
                copy_p = (cs_p["ms_d2h"] + cs_p["ms_h2d"]) / steps
                exp_p = max(0.0, ms - ms_none)
                entry[name] = {
                    "rows": rows, "alpha": [round(r / n, 4) for r, n in zip(rows, lens)],
                    "ms_per_step": ms, "ms_steps": [round(x, 2) for x in alt[name]["steps"]],
                    "tflops": flops["total"] / (ms * 1e-3) / 1e12,
                    "bytes_d2h_per_step": cs_p["bytes_d2h"] / steps, "copy_ms_per_step": copy_p,
                    "exposed_ms_per_step": exp_p,
                    "hidden_pct": 100.0 * max(0.0, min(1.0, 1.0 - exp_p / copy_p)) if copy_p > 0 else None,
                    "modelled_peak_activation_GiB": modelled_peak_bytes(
                        t_fwd, lens, rows, copy_row, freed_row, bw_GBps) / 2**30,
                    "device_memory": device_memory(walks[name], o)}
            for w in walks.values():
                w.close()
            result[part] = entry
            print(f"[bench] policy {part}: full {entry['full']['ms_per_step']:.1f} ms, "
                  f"plan {entry['plan']['ms_per_step']:.1f} ms", file=sys.stderr, flush=True)
        result["all_resident_activation_GiB"] = S * freed_row / 2**30
        result["kv_cache_GiB"] = B * S * 2 * Hkv * D * 2 / 2**30
        return result

    print(f"[bench] workload={args.workload} steps={args.steps} warmup={args.warmup}", file=sys.stderr, flush=True)
    # Headline: exactly K timed steps, no per-kernel events in the stream.
    ms_on, _, cs = timed(ca, args.steps, False)
    steps_on = sorted(step_times[-1])
    print(f"[bench] ms/step={ms_on:.2f}", file=sys.stderr, flush=True)
    # Per-kernel durations for the roofline: K more steps with HIP events
    # around every launch (the events cost a little time, so they are kept
    # out of the headline steps).
    ms_ev, kt, _ = timed(ca, args.steps, True)
    print(f"[bench] ms/step with kernel events={ms_ev:.2f}", file=sys.stderr, flush=True)

    res = {
        "metric": METRIC, "value": None, "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_on, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
    }
    tflops = flops["total"] / (ms_on * 1e-3) / 1e12
    res["value"] = tflops
    res["pct_peak"] = 100.0 * tflops / PEAK_BF16_TFLOPS
    res["ms_per_step_median"] = steps_on[len(steps_on) // 2]
    res["ms_per_step_min"] = steps_on[0]
    res["tokens_per_s"] = S / (ms_on * 1e-3)
    res["config"] = {
        "workload": f"chunked causal attention fwd+bwd, batch {B}, seq {S} in {N} chunks of {S // N}, "
                    f"{Hq} query / {Hkv} KV heads x head_dim {D}, bf16 in / fp32 accumulate, "
                    f"offload {offload} (all chunks but the last), prefetch lookahead {args.lookahead}"
                    + (" (Q/O/LSE offloaded and prefetched back through a device ring; K/V copied to the "
                       "host only, the K/V cache stays resident)" if offload == "qkvol" else ""),
        "name": args.workload, "batch": B, "seq_len": S, "n_chunks": N, "n_q_heads": Hq,
        "n_kv_heads": Hkv, "head_dim": D, "offload": offload,
    }
    steps = args.steps
    res["ms_per_step_with_kernel_events"] = ms_ev
    kern = {}
    for name, v in kt.items():
        per_step = v["ms"] / steps
        k = {"ms_per_step": per_step, "launches_per_step": v["launches"] / steps}
        if flops.get(name):
            k["tflops"] = flops[name] / (per_step * 1e-3) / 1e12
        kern[name] = k
    res["kernels"] = kern
    dom = max((n for n in kern if flops.get(n)), key=lambda n: kern[n]["ms_per_step"])
    ach = kern[dom]["tflops"]
    traffic = measured_traffic(dom, args.workload)
    res["roofline"] = {"kernel": dom, "bound": "mfma", "achieved": ach, "peak": PEAK_BF16_TFLOPS,
                       "unit": "TFLOP/s", "frac": ach / PEAK_BF16_TFLOPS, "traffic": traffic,
                       "traffic_source": (f"profiles/{dom}_{args.workload}_traffic.json: FETCH_SIZE + WRITE_SIZE "
                                          "from separate rocprofv3 --pmc runs of this command, scaled by a 1 GiB "
                                          "copy, kept only while the kernel source's sha256 matches (not "
                                          "measured in this run)") if traffic is not None else None}
    if cs is not None:
        copy_ms = (cs["ms_d2h"] + cs["ms_h2d"]) / steps
        off = {"bytes_d2h_per_step": cs["bytes_d2h"] / steps, "bytes_h2d_per_step": cs["bytes_h2d"] / steps,
               "copy_ms_per_step": copy_ms,
               "d2h_GBps": cs["bytes_d2h"] / max(cs["ms_d2h"], 1e-9) / 1e6,
               "h2d_GBps": cs["bytes_h2d"] / max(cs["ms_h2d"], 1e-9) / 1e6}
        off["kv_copy_only"] = offload == "qkvol"
        if not args.no_offload_compare:
            # The headline walk, the walk that offloads only Q/O/LSE (the set
            # that makes the round trip; in the headline walk K/V are also
            # copied out but never needed back) and the walk that evicts the
            # K/V cache after the forward and streams it back under the last
            # chunk's backward, each timed in alternating steps with the walk
            # without offload, so that clock drift over the run falls on both
            # sides of each comparison alike.
            ca_off = ChunkedAttention(B, S, N, Hq, Hkv, D, dtype="bf16", offload="none")
            alt = {}

            def hidden_of(name):
                a, ms_none = alt[name], alt[name]["ms_none"]
                copy = (a["cs"]["ms_d2h"] + a["cs"]["ms_h2d"]) / steps
                exp = max(0.0, a["ms"] - ms_none)
                return {"ms_per_step": a["ms"], "ms_per_step_no_offload": ms_none,
                        "ms_steps": [round(x, 2) for x in a["steps"]],
                        "ms_steps_no_offload": [round(x, 2) for x in a["steps_none"]],
                        "bytes_d2h_per_step": a["cs"]["bytes_d2h"] / steps,
                        "bytes_h2d_per_step": a["cs"]["bytes_h2d"] / steps, "copy_ms_per_step": copy,
                        "exposed_ms_per_step": exp,
                        "hidden_pct": 100.0 * max(0.0, min(1.0, 1.0 - exp / copy)) if copy > 0 else None}

            # each offloading walk alternates with the walk without offload
            for name in ("offload", "qol", "evict") if offload == "qkvol" else ("offload",):
                w = ca if name == "offload" else ChunkedAttention(
                    B, S, N, Hq, Hkv, D, dtype="bf16", offload={"qol": "qol", "evict": "qkvol_evict"}[name])
                pair = alternate({name: w, "none": ca_off}, steps)
                alt[name] = dict(pair[name], ms_none=pair["none"]["ms"], steps_none=pair["none"]["steps"])
                if w is not ca:
                    w.close()
            head = hidden_of("offload")
            ms_off = head["ms_per_step_no_offload"]
            off["ms_per_step_no_offload"] = ms_off
            off["ms_per_step_offload_alternating"] = head["ms_per_step"]
            off["exposed_ms_per_step"] = head["exposed_ms_per_step"]
            off["hidden_pct"] = head["hidden_pct"]
            if offload == "qkvol":
                off["round_trip_qol"] = hidden_of("qol")
                off["evict"] = hidden_of("evict")
            mem_on = device_memory(ca, out)
            print(f"[bench] device memory with offload: {mem_on['walk_peak_GiB']:.3f} GiB", file=sys.stderr, flush=True)
            mem_off = device_memory(ca_off, out)
            print(f"[bench] device memory without: {mem_off['walk_peak_GiB']:.3f} GiB", file=sys.stderr, flush=True)
            off["device_memory"] = {"offload": mem_on, "no_offload": mem_off}
            off["device_memory"]["saved_GiB"] = (off["device_memory"]["no_offload"]["walk_peak_GiB"] -
                                                 off["device_memory"]["offload"]["walk_peak_GiB"])
            # Per-chunk exposed time: one more step of each with an event at
            # every chunk boundary; exposed = duration with offload minus
            # duration without, per forward and per backward chunk.
            spans = {}
            for name, c in (("on", ca), ("off", ca_off)):
                marks = []
                c.step(inp, out, lookahead=args.lookahead, marks=marks)
                torch.cuda.synchronize()
                spans[name] = {marks[n][0]: marks[n][1].elapsed_time(marks[n + 1][1]) for n in range(len(marks) - 1)}
                print(f"[bench] marked step ({name})", file=sys.stderr, flush=True)
            off["per_chunk_exposed_ms"] = {
                ph: [round(spans["on"][(ph, i)] - spans["off"][(ph, i)], 3) for i in range(N)] for ph in ("fwd", "bwd")}
            ca_off.close()
        # Host-link rates of the library's copy path with nothing else
        # running (1 GiB each way, and both ways at once); T_copy_iso is the
        # step's copy volume at those rates.
        link = L.sppo_link_probe(ca.ctx, 1 << 30)
        iso_ms = (cs["bytes_d2h"] / link["d2h_GBps"] + cs["bytes_h2d"] / link["h2d_GBps"]) / 1e6 / steps
        off["link"] = link
        off["copy_iso_ms_per_step"] = iso_ms
        if "exposed_ms_per_step" in off:
            off["hidden_pct_vs_iso"] = 100.0 * max(0.0, min(1.0, 1.0 - off["exposed_ms_per_step"] / iso_ms))
        res["offload"] = off
        res["offload_hidden_pct"] = off.get("hidden_pct")
        if offload == "qkvol" and not args.no_policy:
            res["offload_policy"] = policy_compare(link["d2h_GBps"])
    ca.close()
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle sample", file=sys.stderr, flush=True)
        cb = oracle_cpu_baseline(inp, D, args.cpu_sample_tokens, args.cpu_sample_heads)
        res["cpu_baseline"] = {k: cb[k] for k in ("value", "unit", "cores", "kind", "sample", "affinity_cpus")}
        res["cpu_baseline"]["cpu_model"] = cpu_model()
        # an extrapolation from the measured rate, not a measurement
        res["cpu_baseline"]["extrapolated_full_step_s"] = flops["total"] / (cb["value"] * 1e12)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
