"""Throughput of the full K-VEC prefill eviction step on one MI355X.

One step = window scores for every layer, then the coverage-aware selection
of every layer in order (each layer reads the coverage bitmap of the earlier
ones) and the gather of the kept K/V into the compacted cache: every stage of
the hot path, on synthetic Llama-3.1-8B-shaped inputs resident in HBM.

Prints one JSON line: prefix tokens/s (batch * T per step / step time), the
roofline of the dominant kernel (live HIP-event timing), and the CPU oracle
timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
MFMA_BF16_PEAK_TFLOPS = 2500.0  # dense bf16


def _hip():
    lib = ctypes.CDLL("libamdhip64.so")
    lib.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
    lib.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                        ctypes.c_void_p]
    lib.hipEventDestroy.argtypes = [ctypes.c_void_p]
    lib.hipEventSynchronize.argtypes = [ctypes.c_void_p]
    lib.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    return lib


def _events(hip, n):
    out = []
    for _ in range(n):
        e = ctypes.c_void_p()
        assert hip.hipEventCreate(ctypes.byref(e)) == 0
        out.append(e.value)
    return out


def _elapsed(hip, a, b) -> float:
    ms = ctypes.c_float()
    assert hip.hipEventElapsedTime(ctypes.byref(ms), a, b) == 0
    return ms.value


def cpu_baseline(w, max_layers: int, min_seconds: float = 10.0):
    """The C++ oracle as it stands, timed on sequence 0 layer by layer in the
    step's order (layer l uses the bitmaps of layers < l), until about
    `min_seconds` of oracle work or `max_layers` layer evictions.  Its window
    scores (the dominant part) run on every CPU this process may use; the
    policy steps and the gather are single-threaded."""
    import numpy as np

    import synth
    from oracle import cxx
    threads = cxx.default_threads()
    t_work = 0.0
    done = 0
    prev = []
    while done < max_layers and (done == 0 or t_work < min_seconds):
        l = done % w.n_layers
        if l == 0:
            prev = []
        q = synth.to_f64(synth.queries(w, l, 0), w.dtype)
        k = synth.to_f64(synth.keys(w, l, 0), w.dtype)
        v = synth.values(w, l, 0)
        t0 = time.perf_counter()
        p, pe, imp = cxx.score_layer(q, k, w.window, threads=threads)
        n_t = cxx.counts_from_bits(prev) if prev else np.zeros(w.seq_len, np.int64)
        res = cxx.evict_layer_from_scores(p, pe, imp, n_t, l, w)
        cxx.gather_rows(k, res.idx)
        cxx.gather_rows(v, res.idx)
        t_work += time.perf_counter() - t0
        prev.append(res.bits)
        done += 1
    per_layer = t_work / done
    step_s = per_layer * w.n_layers * w.batch
    return {"value": w.batch * w.seq_len / step_s, "unit": "prefix tokens/s",
            "cores": threads, "host_cpus": len(os.sched_getaffinity(0)),
            "kind": "oracle", "impl": "C++ (oracle/kvec_oracle.cpp), float64 window scores on "
                                      f"{threads} threads",
            "sample": f"{done} layer evictions of sequence 0 in layer order ({t_work:.1f} s of "
                      f"oracle work, input generation excluded); per-layer time extrapolated "
                      f"to {w.n_layers} layers x batch {w.batch}"}


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "step_kernel_{workload}_traffic.md")
SOURCE_DIRS = (os.path.join(ROOT, "paper_2606_29563_amd", "csrc"), os.path.join(ROOT, "include"))
# sources outside the step kernel's build (they do not change its counters)
DIGEST_SKIP = ("kvec_decode.hip",)


def source_digest() -> str:
    """sha256 over the HIP sources and headers the kernels are built from."""
    import hashlib
    h = hashlib.sha256()
    for d in SOURCE_DIRS:
        for name in sorted(os.listdir(d)):
            if name.endswith((".hip", ".h")) and name not in DIGEST_SKIP:
                h.update(name.encode())
                with open(os.path.join(d, name), "rb") as f:
                    h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(workload: str):
    """HBM bytes per fused launch from the committed counter summary, or None
    when there is none or the kernel sources changed since it was taken."""
    path = TRAFFIC_FILE.format(workload=workload)
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as f:
        for line in f:
            if line.startswith("- ") and " = " in line:
                k, v = line[2:].split(" = ", 1)
                vals[k.strip()] = v.strip().strip("`")
    if vals.get("source_digest") != source_digest():
        return None
    try:
        return int(vals["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def prefill_lse(q, k, w):
    """The window rows' log-sum-exp that the layer's prefill attention hands over
    (input preparation for kvec_evict_model_lse, not timed): fp32 causal
    logsumexp of q . k / sqrt(d) over keys 0..p of each window row, with torch
    on the device.  Returns [L][b][HQ][Wn] fp32."""
    import math

    import torch
    L, b, HQ, Wn, d = q.shape
    G = HQ // k.shape[2]
    T = k.shape[3]
    pos = T - Wn + torch.arange(Wn, device=q.device)
    hidden = torch.arange(T, device=q.device)[None, :] > pos[:, None]     # [Wn][T]
    out = torch.empty((L, b, HQ, Wn), dtype=torch.float32, device=q.device)
    for l in range(L):
        for s in range(b):
            kt = k[l, s].float().transpose(1, 2).contiguous()              # [H][d][T]
            for j0 in range(0, HQ, G):
                qs = q[l, s, j0:j0 + G].float()                             # [G][Wn][d]
                lg = torch.matmul(qs, kt[j0 // G]) / math.sqrt(d)            # [G][Wn][T]
                lg.masked_fill_(hidden, float("-inf"))
                out[l, s, j0:j0 + G] = torch.logsumexp(lg, dim=-1)
    return out


def time_steps(hip, stream, run, steps: int, warmup: int):
    """Per-step durations (ms) between HIP events at the step boundaries, and
    the host wall time (ms) of the timed steps."""
    import torch
    evs = _events(hip, steps + 1)
    for _ in range(warmup):
        run()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    # events only between steps: a record between launches adds a few us of
    # gap to each of them
    assert hip.hipEventRecord(evs[0], stream) == 0
    for s in range(steps):
        run()
        assert hip.hipEventRecord(evs[s + 1], stream) == 0
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) * 1e3
    durs = [_elapsed(hip, evs[s], evs[s + 1]) for s in range(steps)]
    for e in evs:
        hip.hipEventDestroy(e)
    return durs, wall


def stage_breakdown(hip, stream, w, cfg, q, k, v, ws, idx, ko, vo, args) -> None:
    """Per-layer entry points of every layer in order, each call bracketed by
    HIP events: the separate launches of the score passes, the selection and
    the gather (the fused step overlaps them; this shows each one's rate)."""
    import torch
    L, b, H, HQ, T, d, B = (w.n_layers, w.batch, w.n_kv_heads, w.n_q_heads, w.seq_len,
                            w.head_dim, w.budget)
    es = 2 if w.dtype == "bf16" else 4
    Tc = w.candidates
    p = torch.empty((b, H, Tc), dtype=torch.float32, device=q.device)
    pe = torch.empty_like(p)
    imp = torch.empty((b, Tc), dtype=torch.float32, device=q.device)
    bits = torch.zeros((b, L, (T + 63) // 64), dtype=torch.int64, device=q.device)
    calls = {
        "kvec_score": lambda l: kvec_mod().kvec_score(cfg, q[l], k[l], p, pe, imp, ws),
        "kvec_select_cover": lambda l: kvec_mod().kvec_select_cover(cfg, l, p, pe, imp, bits,
                                                                    idx[l], None, ws),
        "kvec_compact": lambda l: kvec_mod().kvec_compact(cfg, k[l], v[l], idx[l], ko[l], vo[l]),
    }
    for _ in range(max(1, args.warmup)):
        for l in range(L):
            for fn in calls.values():
                fn(l)
    torch.cuda.synchronize()
    evs = _events(hip, 2 * L * len(calls))
    for l in range(L):
        for i, fn in enumerate(calls.values()):
            e = 2 * (l * len(calls) + i)
            assert hip.hipEventRecord(evs[e], stream) == 0
            fn(l)
            assert hip.hipEventRecord(evs[e + 1], stream) == 0
    torch.cuda.synchronize()
    out = {}
    # bytes each call must move at least: the keys once and the query window
    # (scores), the scores and counts (selection), the kept rows read and
    # written (gather)
    need = {"kvec_score": b * (H * T * d * es + HQ * w.rows * d * es + (2 * H + 1) * Tc * 4),
            "kvec_select_cover": b * ((2 * H + 1) * Tc * 4 + H * B * 4),
            "kvec_compact": b * 4 * H * B * d * es}
    for i, name in enumerate(calls):
        us = [_elapsed(hip, evs[2 * (l * len(calls) + i)], evs[2 * (l * len(calls) + i) + 1]) * 1e3
              for l in range(L)]
        avg = sum(us) / len(us)
        gbs = need[name] / (avg * 1e-6) / 1e9
        out[name] = {"us_per_layer": round(avg, 2), "algorithmic_bytes": need[name],
                     "achieved_GBps": round(gbs, 1), "hbm_frac": round(gbs / HBM_PEAK_GBS, 4)}
    print(json.dumps({"workload": w.name, "mode": "per-layer entry points", "stages": out}))


def ms_lse_of(obj) -> float:
    return obj["ms_per_step"]


def kvec_mod():
    from paper_2606_29563_amd import kvec
    return kvec


def copy_calibration(mib: int) -> None:
    """A plain device copy of known size, to scale the HBM byte counters."""
    import torch
    n = mib << 20
    src = torch.ones(n, dtype=torch.uint8, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": n, "copies": 3}))


def gen_inputs(w, dev, dt, n_gen=None):
    """Device tensors q [L][b][HQ][O'][d], k and v [L][b][H][T][d] of a synthetic
    workload.  With n_gen < L only layers 0..n_gen-1 are generated and layer l
    holds a copy of layer l % n_gen (separate device memory)."""
    import torch

    import synth
    L, b, H, HQ, T, d = w.n_layers, w.batch, w.n_kv_heads, w.n_q_heads, w.seq_len, w.head_dim
    n_gen = L if n_gen is None else min(n_gen, L)
    q = torch.empty((L, b, HQ, w.rows, d), dtype=dt, device=dev)
    k = torch.empty((L, b, H, T, d), dtype=dt, device=dev)
    v = torch.empty_like(k)
    for l in range(n_gen):
        for s in range(b):
            for dst, arr in ((q, synth.queries(w, l, s)), (k, synth.keys(w, l, s)),
                             (v, synth.values(w, l, s))):
                t = torch.from_numpy(arr)
                if w.dtype == "bf16":
                    t = t.view(torch.bfloat16)
                dst[l, s].copy_(t)
    for l in range(n_gen, L):
        for x in (q, k, v):
            x[l].copy_(x[l % n_gen])
    return q, k, v


def measure_other(wi, args, hip, stream):
    """One more workload, timed like the headline: the isolated step (K steps,
    one call each) and K pipelined steps in one call.  The fractions are the
    step's algorithmic bytes and flops (as for the headline) over the step's
    GPU time between HIP events."""
    import torch

    import synth
    from paper_2606_29563_amd import kvec
    w = synth.workload(wi)
    dev = torch.device("cuda:0")
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    L, b, H, HQ, T, d, B = (w.n_layers, w.batch, w.n_kv_heads, w.n_q_heads, w.seq_len,
                            w.head_dim, w.budget)
    # the large prefixes generate 4 layers and repeat them (the step's cost does
    # not depend on which layer's values it reads, only on their distribution)
    n_gen = L if b * T <= 32768 else 4
    print(f"[bench] other workload {w.name}: generating {n_gen} of {L} layers", file=sys.stderr,
          flush=True)
    q, k, v = gen_inputs(w, dev, dt, n_gen)
    cfg = kvec.Config.from_workload(w)
    ws = torch.empty(kvec.kvec_workspace_size(cfg), dtype=torch.uint8, device=dev)
    bits = torch.empty((b, L, (T + 63) // 64), dtype=torch.int64, device=dev)
    idx = torch.empty((L, b, H, B), dtype=torch.int32, device=dev)
    ko = torch.empty((L, b, H, B, d), dtype=dt, device=dev)
    vo = torch.empty_like(ko)
    es = 2 if w.dtype == "bf16" else 4
    step_bytes = L * b * (H * T * d * es + HQ * w.rows * d * es + 4 * H * B * d * es)
    O, Wn, delta = w.window, w.rows, w.n_adjust_heads if w.rows > w.window else 0
    step_flops = 2 * d * L * b * (HQ * O * T + (HQ // H) * delta * (Wn - O) * T)
    durs, wall = time_steps(hip, stream,
                            lambda: kvec.kvec_evict_model(cfg, q, k, v, bits, idx, ko, vo, ws),
                            args.steps, args.warmup)
    ms = wall / args.steps
    ms_gpu = sum(durs) / len(durs)
    n = max(2, args.steps)
    bn = torch.empty((n,) + tuple(bits.shape), dtype=bits.dtype, device=dev)
    iN = torch.empty((n,) + tuple(idx.shape), dtype=idx.dtype, device=dev)
    kon = torch.empty((n,) + tuple(ko.shape), dtype=ko.dtype, device=dev)
    von = torch.empty_like(kon)
    qn, kn, vn = (x.unsqueeze(0).expand(n, *x.shape) for x in (q, k, v))
    durs, _ = time_steps(hip, stream,
                         lambda: kvec.kvec_evict_model_steps(cfg, qn, kn, vn, bn, iN, kon, von, ws), 2, 1)
    assert all(torch.equal(iN[i], idx) for i in range(n)), "pipelined steps differ"
    ms_pipe = sum(durs) / len(durs) / n
    out = {"workload": w.name, "layers": L, "batch": b, "kv_heads": H, "q_heads": HQ,
           "seq_len": T, "budget": B, "generated_layers": n_gen, "ms_per_step": round(ms, 4),
           "value": round(b * T / (ms * 1e-3), 1), "unit": "prefix tokens/s",
           "hbm_frac": round(step_bytes / (ms_gpu * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
           "mfma_frac": round(step_flops / (ms_gpu * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4),
           "pipelined_ms_per_step": round(ms_pipe, 4),
           "pipelined_value": round(b * T / (ms_pipe * 1e-3), 1)}
    print(f"[bench] {w.name}: {ms:.4f} ms per step, pipelined {ms_pipe:.4f}", file=sys.stderr,
          flush=True)
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", type=int, default=2, help="index of the synthetic workload")
    ap.add_argument("--cpu-sample-layers", type=int, default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--path", choices=("both", "model", "lse"), default="both",
                    help="model: kvec_evict_model only; lse: kvec_evict_model_lse only "
                         "(row normalisers from the prefill); both: the headline plus the "
                         "given-lse step as a second object")
    ap.add_argument("--stages", action="store_true",
                    help="instead of the step: the per-layer entry points (kvec_score, "
                         "kvec_select_cover, kvec_compact) one by one, each timed on its own")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB (counter calibration)")
    ap.add_argument("--other-workloads", default=None, metavar="LIST",
                    help="comma-separated workload indices also measured (isolated and "
                         "pipelined step) and reported under other_workloads; default 1,3,4,5 "
                         "for the headline run, empty to skip")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU; multi-GPU runs are not part of this build "
              f"(asked for --gpus {args.gpus})", file=sys.stderr)
        sys.exit(2)
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return

    import torch

    import synth
    from paper_2606_29563_amd import kvec

    w = synth.workload(args.workload)
    kvec.load()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    L, b, H, HQ, T, d, B = (w.n_layers, w.batch, w.n_kv_heads, w.n_q_heads, w.seq_len,
                            w.head_dim, w.budget)
    print(f"[bench] {w.name}: generating {L} layers of inputs", file=sys.stderr, flush=True)
    q, k, v = gen_inputs(w, dev, dt)
    cfg = kvec.Config.from_workload(w)
    ws = torch.empty(kvec.kvec_workspace_size(cfg), dtype=torch.uint8, device=dev)
    bits = torch.empty((b, L, (T + 63) // 64), dtype=torch.int64, device=dev)
    idx = torch.empty((L, b, H, B), dtype=torch.int32, device=dev)
    ko = torch.empty((L, b, H, B, d), dtype=dt, device=dev)
    vo = torch.empty_like(ko)
    torch.cuda.synchronize()
    print("[bench] inputs resident; warming up", file=sys.stderr, flush=True)

    hip = _hip()
    stream = torch.cuda.current_stream().cuda_stream  # the library's stream
    if args.stages:
        stage_breakdown(hip, stream, w, cfg, q, k, v, ws, idx, ko, vo, args)
        return
    es = 2 if w.dtype == "bf16" else 4
    # algorithmic bytes of the whole step: K read once, the Q window, the gather
    # (read and write of the kept K and V rows)
    step_bytes = L * b * (H * T * d * es + HQ * w.rows * d * es + 4 * H * B * d * es)
    tokens = b * T

    # algorithmic MFMA work of the whole step: the last-O rows of every query
    # head and the extended rows of the G query heads of the delta H_top heads,
    # over every key of the prefix
    O, Wn, delta = w.window, w.rows, w.n_adjust_heads if w.rows > w.window else 0
    step_flops = 2 * d * L * b * (HQ * O * T + (HQ // H) * delta * (Wn - O) * T)

    def mfma(ms_step_gpu, passes):
        # frac: the method's own matrix work (one product per logit) over the
        # step time; executed_*: what the kernel runs (one product per score
        # pass, two when the row normalisers are computed here)
        tf = step_flops / (ms_step_gpu * 1e-3) / 1e12
        tx = step_flops * passes / (ms_step_gpu * 1e-3) / 1e12
        return {"bound": "mfma", "achieved": round(tf, 1), "peak": MFMA_BF16_PEAK_TFLOPS,
                "unit": "TFLOP/s", "frac": round(tf / MFMA_BF16_PEAK_TFLOPS, 4),
                "flops_per_step": step_flops,
                "executed_passes": passes, "executed_flops_per_step": step_flops * passes,
                "executed_achieved": round(tx, 1),
                "executed_frac": round(tx / MFMA_BF16_PEAK_TFLOPS, 4),
                "note": "algorithmic flops: one q.k product per logit of the last-O rows of "
                        "every query head and of the extended rows of the H_top heads; dense "
                        "bf16 peak"}

    def roofline(durs, n_launch, traffic):
        # Average duration of a fused launch: each step's interval between HIP
        # events on the library's stream, over its launches (the few-us gaps
        # between dispatches included).  In the steady state a launch does one
        # layer's worth of every stage of the layer pipeline.
        avg_ms = sum(durs) / len(durs) / n_launch
        per_launch = step_bytes / n_launch
        achieved = per_launch / (avg_ms * 1e-3) / 1e9
        return {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                "kernel": "step_kernel (fused pipeline launch)", "launches_per_step": n_launch,
                "avg_launch_us": round(avg_ms * 1e3, 2),
                "algorithmic_bytes_per_launch": int(per_launch)}

    roof = ms_step = mfma_obj = None
    if args.path in ("both", "model"):
        n_launch = kvec.kvec_profile_points(cfg) - 1
        durs, wall = time_steps(
            hip, stream, lambda: kvec.kvec_evict_model(cfg, q, k, v, bits, idx, ko, vo, ws),
            args.steps, args.warmup)
        ms_step = wall / args.steps
        print(f"[bench] {args.steps} steps in {wall:.2f} ms", file=sys.stderr, flush=True)
        roof = roofline(durs, n_launch, measured_traffic(w.name))
        mfma_obj = mfma(sum(durs) / len(durs), 2)

    dec_obj = None
    if args.path == "both":
        try:
            # Decode attention over the compacted cache of the last step: one new
            # token, every layer (the consumer of the cache the step writes).
            g = torch.Generator().manual_seed(77)
            qd = torch.randn((L, b, HQ, d), generator=g).to(dt).to(dev)
            outd = torch.empty((L, b, HQ, d), dtype=torch.float32, device=dev)
            wsd = torch.empty(kvec.kvec_decode_workspace_size(cfg, B), dtype=torch.uint8, device=dev)

            def decode_all():
                for l in range(L):
                    kvec.kvec_decode_attention(cfg, qd[l], ko[l], vo[l], outd[l], wsd, idx=idx[l])

            durs, _ = time_steps(hip, stream, decode_all, max(args.steps, 20), args.warmup)
            us_eager = sum(durs) / len(durs) / L * 1e3
            # The per-layer calls issued from Python are host-bound; the GPU time
            # comes from replaying the same L calls captured in a HIP graph (no
            # memset nodes), each replay checked against the eager result.
            want = outd.clone()
            graph = torch.cuda.CUDAGraph()
            side = torch.cuda.Stream()
            side.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(side):
                decode_all()
            torch.cuda.current_stream().wait_stream(side)
            with torch.cuda.graph(graph):
                decode_all()
            for _ in range(3):
                outd.zero_()
                graph.replay()
                torch.cuda.synchronize()
                assert torch.equal(outd, want), "graph replay differs from the eager decode"
            reps = max(args.steps, 20)
            gdurs, _ = time_steps(hip, stream, graph.replay, reps, 2)
            us = sum(gdurs) / len(gdurs) / L * 1e3
            dbytes = b * (2 * H * B * d * es + HQ * d * es + HQ * d * 4 + H * B * 4)
            dec_obj = {"entry": "kvec_decode_attention",
                       "what": "one decode token's attention over the compacted cache, per layer "
                               "(two launches: partial chunks, combine); GPU time of the L calls "
                               "replayed from a HIP graph",
                       "us_per_layer": round(us, 2), "us_per_layer_python_issue": round(us_eager, 2),
                       "cache_rows": B,
                       "roofline": {"bound": "hbm", "achieved": round(dbytes / (us * 1e-6) / 1e9, 1),
                                    "peak": HBM_PEAK_GBS, "unit": "GB/s",
                                    "frac": round(dbytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
                                    "algorithmic_bytes_per_call": dbytes}}
            print(f"[bench] decode attention: {us:.2f} us per layer", file=sys.stderr, flush=True)
        except Exception as e:  # the headline line must not depend on this extra
            dec_obj = {"entry": "kvec_decode_attention", "error": repr(e)}
            print(f"[bench] decode attention failed: {e!r}", file=sys.stderr, flush=True)

    lse_obj = None

    def measure_lse():
        print("[bench] window-row log-sum-exp (prefill attention stand-in)", file=sys.stderr,
              flush=True)
        lse = prefill_lse(q, k, w)
        n_launch = kvec.kvec_profile_points_lse(cfg) - 1
        durs, wall = time_steps(
            hip, stream,
            lambda: kvec.kvec_evict_model_lse(cfg, q, lse, k, v, bits, idx, ko, vo, ws),
            args.steps, args.warmup)
        print(f"[bench] given-lse: {args.steps} steps in {wall:.2f} ms", file=sys.stderr,
              flush=True)
        ms_lse = wall / args.steps
        lse_obj = {"entry": "kvec_evict_model_lse",
                   "what": "the same step with the window rows' log-sum-exp handed over by the "
                           "layer's prefill attention (one score pass over K instead of two)",
                   "value": round(tokens / (ms_lse * 1e-3), 1), "unit": "prefix tokens/s",
                   "ms_per_step": round(ms_lse, 4),
                   "roofline": roofline(durs, n_launch, measured_traffic(w.name + "-lse")),
                   "mfma_roofline": mfma(sum(durs) / len(durs), 1)}
        if args.path != "both":  # profiled runs time the isolated step only
            return lse_obj
        try:
            # n back-to-back steps in one call (kvec_evict_model_lse_steps),
            # inputs and normalisers with step stride 0, n distinct outputs
            n = max(2, args.steps)
            qn, kn, vn, ln = (x.unsqueeze(0).expand(n, *x.shape) for x in (q, k, v, lse))
            bn = torch.empty((n,) + tuple(bits.shape), dtype=bits.dtype, device=dev)
            iN = torch.empty((n,) + tuple(idx.shape), dtype=idx.dtype, device=dev)
            kon = torch.empty((n,) + tuple(ko.shape), dtype=ko.dtype, device=dev)
            von = torch.empty_like(kon)
            pd, _ = time_steps(
                hip, stream,
                lambda: kvec.kvec_evict_model_lse_steps(cfg, qn, ln, kn, vn, bn, iN, kon, von, ws),
                3, 1)
            assert all(torch.equal(iN[i], idx) for i in range(n)), "pipelined steps differ"
            ms_pipe = sum(pd) / len(pd) / n
            ach = step_bytes / (ms_pipe * 1e-3) / 1e9
            lse_obj["pipelined_steps"] = {
                "entry": "kvec_evict_model_lse_steps", "steps_per_call": n,
                "value": round(tokens / (ms_pipe * 1e-3), 1), "unit": "prefix tokens/s",
                "ms_per_step": round(ms_pipe, 4),
                "roofline": {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS,
                             "unit": "GB/s", "frac": round(ach / HBM_PEAK_GBS, 4)},
                "mfma_roofline": mfma(ms_pipe, 1)}
            print(f"[bench] given-lse pipelined: {ms_pipe:.4f} ms per step", file=sys.stderr,
                  flush=True)
            del bn, iN, kon, von
        except Exception as e:  # the given-lse object must not depend on this extra
            lse_obj["pipelined_steps"] = {"entry": "kvec_evict_model_lse_steps", "error": repr(e)}
            print(f"[bench] given-lse pipelined steps failed: {e!r}", file=sys.stderr, flush=True)
        return lse_obj

    if args.path == "lse":
        lse_obj = measure_lse()
        roof, ms_step, mfma_obj = lse_obj["roofline"], ms_lse_of(lse_obj), lse_obj["mfma_roofline"]
    elif args.path == "both":
        try:
            lse_obj = measure_lse()
        except Exception as e:  # the headline line must not depend on this extra
            lse_obj = {"entry": "kvec_evict_model_lse", "error": repr(e)}
            print(f"[bench] given-lse step failed: {e!r}", file=sys.stderr, flush=True)

    steps_obj = None
    if args.path == "both":
        # The same step for n back-to-back prefills in one call
        # (kvec_evict_model_steps): one layer pipeline over the n x L layers,
        # so each step's closing launches overlap the next one's opening.
        # Inputs: the resident prefill, evicted n times (step stride 0);
        # outputs: n distinct sets.  Reported beside the headline, which is
        # one isolated step per call.
        try:
            n = max(2, args.steps)
            print(f"[bench] {n} pipelined steps per call", file=sys.stderr, flush=True)
            qn = q.unsqueeze(0).expand(n, *q.shape)
            kn = k.unsqueeze(0).expand(n, *k.shape)
            vn = v.unsqueeze(0).expand(n, *v.shape)
            bn = torch.empty((n,) + tuple(bits.shape), dtype=bits.dtype, device=dev)
            iN = torch.empty((n,) + tuple(idx.shape), dtype=idx.dtype, device=dev)
            kon = torch.empty((n,) + tuple(ko.shape), dtype=ko.dtype, device=dev)
            von = torch.empty_like(kon)
            reps = 3
            durs, wall = time_steps(
                hip, stream, lambda: kvec.kvec_evict_model_steps(cfg, qn, kn, vn, bn, iN, kon, von, ws),
                reps, 1)
            # every step's indices equal those of one isolated step
            kvec.kvec_evict_model(cfg, q, k, v, bits, idx, ko, vo, ws)
            torch.cuda.synchronize()
            assert all(torch.equal(iN[i], idx) for i in range(n)), "pipelined steps differ"
            ms_pipe = sum(durs) / len(durs) / n
            ach = step_bytes / (ms_pipe * 1e-3) / 1e9
            steps_obj = {"entry": "kvec_evict_model_steps", "steps_per_call": n,
                         "what": "n back-to-back prefills evicted in one call: one layer pipeline "
                                 "over their n x L layers (n x L + 11 fused launches)",
                         "inputs": "the resident prefill for every step (step stride 0); "
                                   "n distinct output sets",
                         "value": round(tokens / (ms_pipe * 1e-3), 1), "unit": "prefix tokens/s",
                         "ms_per_step": round(ms_pipe, 4),
                         "roofline": {"bound": "hbm", "achieved": round(ach, 1),
                                      "peak": HBM_PEAK_GBS, "unit": "GB/s",
                                      "frac": round(ach / HBM_PEAK_GBS, 4)},
                         "mfma_roofline": mfma(ms_pipe, 2)}
            del bn, iN, kon, von
            print(f"[bench] pipelined: {ms_pipe:.4f} ms per step", file=sys.stderr, flush=True)
        except Exception as e:  # the headline line must not depend on this extra
            steps_obj = {"entry": "kvec_evict_model_steps", "error": repr(e)}
            print(f"[bench] pipelined steps failed: {e!r}", file=sys.stderr, flush=True)

    others = None
    ow = args.other_workloads
    if ow is None:
        ow = "1,3,4,5" if (args.workload == 2 and args.path == "both") else ""
    if ow:
        others = []
        for wi in [int(x) for x in ow.split(",") if x.strip()]:
            try:
                others.append(measure_other(wi, args, hip, stream))
            except Exception as e:  # the headline line must not depend on this extra
                others.append({"workload_index": wi, "error": repr(e)})
                print(f"[bench] workload {wi} failed: {e!r}", file=sys.stderr, flush=True)
            torch.cuda.empty_cache()

    cpu = None
    if not args.no_cpu_baseline:
        # layers of sequence 0 in order until about 10 s of oracle work
        sample = args.cpu_sample_layers or 4 * L
        print(f"[bench] CPU oracle on {sample} layer(s)", file=sys.stderr, flush=True)
        cpu = cpu_baseline(w, sample)

    out = {
        "metric": "prefix tokens/s through full eviction step (all layers); % HBM/MFMA roofline",
        "value": round(tokens / (ms_step * 1e-3), 1), "unit": "prefix tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": w.name, "layers": L, "batch": b, "kv_heads": H, "q_heads": HQ,
                   "head_dim": d, "seq_len": T, "window": w.window, "window_ext": w.window_ext,
                   "budget": B, "pool": w.pool_kernel, "delta": w.n_adjust_heads,
                   "lambda": w.lam, "beta": w.beta, "head_criterion": w.criterion},
        "roofline": roof,
        "mfma_roofline": mfma_obj,
        "cpu_baseline": cpu,
    }
    if args.path == "lse":
        out["config"]["entry"] = "kvec_evict_model_lse"
    elif lse_obj is not None:
        out["prefill_lse_step"] = lse_obj
    if steps_obj is not None:
        out["pipelined_steps"] = steps_obj
    if others is not None:
        out["other_workloads"] = others
    if dec_obj is not None:
        out["decode_attention"] = dec_obj
    print(json.dumps(out))


if __name__ == "__main__":
    main()
