#!/usr/bin/env python3
"""Benchmark of the decode-attention hot path on one MI355X.

One step = one pass of the whole path over one batch: KV append (every KV
head of every sequence gets one new row) followed by decode attention of
every query head -- run as the fused step, two kernels: the partial kernel
(which also performs the append) and the merge (which also advances len);
this is da_decode_step, called as its two halves so that events can bracket
the partial kernel in a second pass over the same steps (a step that
da_decode_step runs as one launch, on short slabs, is timed whole there).
The timed region itself holds only the K steps' launches: an event recorded
between two launches delays the second.  The default workload is
the long-context ragged GQA configuration (B=4, h_q=64, h_kv=8, d=128,
len ~ U{65536..131008}, n_max=131072, 64 append+decode steps).

Prints ONE JSON line:
  value        algorithmic HBM bytes of the step (paper's traffic model:
               K/V rows read once per KV head over len_b rows, q read and
               output written once per query head, the appended rows) divided
               by the measured time per step, in GB/s; inputs are resident in
               HBM before the timed region starts.
  roofline     the dominant kernel (decode_partial_kernel): its algorithmic
               bytes per launch over its average launch duration, measured with
               HIP events on the stream it runs on (in the second pass over the
               same K steps), against the 8 TB/s HBM peak;
               `traffic` = HBM bytes per launch from rocprofv3 FETCH_SIZE and
               WRITE_SIZE counters (profiles/decode_partial_counters.json),
               null when the kernel source changed since they were taken;
               `ceiling` = a plain streaming read of the same K and V
               allocations on this machine (the practical read ceiling) and
               the partial kernel's bandwidth as a fraction of it.
  cpu_baseline the CPU oracle (plain fp64 loops, OpenMP over heads) timed on
               this host on a bounded sample of the same workload.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload c5]
                       [--graph]   (replay the timed steps as one HIP graph)
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

METRIC = "achieved HBM GB/s and µs per decode step (fp32 GQA), % of HBM roofline"
HBM_PEAK_GBPS = 8000.0
KERNEL_SRC = os.path.join(ROOT, "paper_2607_19456_amd", "csrc", "decode_attn.hip")
COUNTERS = os.path.join(ROOT, "profiles", "decode_partial_counters.json")


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kernel_build_hash() -> str:
    """sha256 of the kernel source and the compiler flags it is built with
    (either changes the code the counters were taken on).  Paths in the
    flags are taken relative to the repository, so the hash does not depend
    on where the checkout lives."""
    from paper_2607_19456_amd import build
    with open(KERNEL_SRC, "rb") as f:
        src = f.read()
    flags = ["-I" + os.path.relpath(f[2:], ROOT) if f.startswith("-I") else f
             for f in build.FLAGS]
    return hashlib.sha256(src + "\n".join(flags).encode()).hexdigest()


def counter_traffic(workload: str):
    """HBM bytes per decode_partial launch from the committed counter runs,
    or None when they are absent, for another workload, or stale."""
    try:
        with open(COUNTERS) as f:
            c = json.load(f)
    except (OSError, ValueError):
        return None
    if c.get("kernel_build_sha256") != kernel_build_hash() or c.get("workload") != workload:
        return None
    return c.get("hbm_bytes_per_launch")


def custom_shape(spec: str):
    """A workload from 'key=value,...' (keys of workloads.custom)."""
    from paper_2607_19456_amd import workloads

    kw = {}
    for item in spec.split(","):
        key, _, val = item.partition("=")
        kw[key.strip()] = int(val)
    steps, rows = kw.get("steps", 0), kw.get("rows", 1)
    if "len_lo" not in kw:
        kw["len_lo"] = max(1, kw["n_max"] - steps * rows)
    kw.setdefault("len_hi", kw["len_lo"])
    name = ("custom_B{B}_hq{h_q}_hkv{h_kv}_dk{d_k}_dv{d_v}_n{n_max}_len{len_lo}-{len_hi}"
            .format(**kw) + (f"_{steps}steps" if steps else "") +
            (f"_x{rows}rows" if rows > 1 else ""))
    return workloads.custom(name, **kw)


def read_ceiling(a, b, stream, reps: int = 5):
    """Mean GB/s of a plain streaming read of device tensors a and b (the
    practical HBM read ceiling on those buffers), and the bytes read."""
    import torch

    from paper_2607_19456_amd import hbm_probe

    nbytes = a.numel() * a.element_size() + b.numel() * b.element_size()
    partial = hbm_probe.read(a, b, stream=stream)
    ms = []
    for _ in range(reps):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        hbm_probe.read(a, b, partial=partial, stream=stream)
        e1.record(stream)
        e1.synchronize()
        ms.append(e0.elapsed_time(e1))
    return nbytes / (sum(ms) / len(ms) * 1e-3) / 1e9, nbytes


def host_cores() -> int:
    """The CPUs this process may run on."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, n)


def cpu_baseline(inp, budget_s: float, step_bytes, gpu_first=None, threads=None):
    """Time the oracle (append + decode of every head, step after step) on
    this host until about budget_s seconds of work are done, with ``threads``
    OpenMP threads (default: every CPU of this process's affinity).  With
    ``gpu_first`` (the GPU's output of the first step, every head), also
    return the max-abs-err between it and the oracle's first step."""
    import numpy as np

    import oracle

    s = inp.shape
    threads = threads or host_cores()
    hK, hV, hl = inp.K, inp.V, inp.lens.copy()
    done, elapsed, nbytes = 0, 0.0, 0
    steps = max(1, s.steps)
    err = None
    while True:
        t = done % steps
        t0 = time.perf_counter()
        if s.rows > 1:
            oracle.append_rows(hK, hV, inp.k_new[t], inp.v_new[t], hl)
            ref = oracle.decode_multi(inp.q_step[t], hK, hV, hl, s.scale32(), threads=threads)
        else:
            if s.steps:
                oracle.append(hK, hV, inp.k_new[t], inp.v_new[t], hl)
                q = inp.q_step[t]
            else:
                q = inp.q
            ref = oracle.decode(q, hK, hV, hl, s.scale32(), threads=threads)
        elapsed += time.perf_counter() - t0
        if done == 0 and gpu_first is not None:
            err = float(np.max(np.abs(gpu_first - ref)))
        nbytes += step_bytes(hl, bool(s.steps))
        done += 1
        log(f"cpu_baseline: oracle step {done} ({elapsed:.1f} s)")
        if elapsed >= budget_s or (s.steps and done >= s.steps):
            break
    return {
        "value": nbytes / elapsed / 1e9,
        "unit": "GB/s",
        "cores": threads,
        "kind": "oracle",
        "sample": (f"{done} full step(s) ({'append + ' if s.steps else ''}decode of all "
                   f"{s.B * s.h_q * s.rows} query rows) of the same workload, {elapsed:.2f} s, "
                   f"fp64 oracle, {threads} OpenMP threads"),
        "seconds_per_step": elapsed / done,
        "cpu_model": _cpu_model(),
        "max_abs_err_first_step": err,
    }


def conventional_leg(s, inp, dev, our_us_per_step, steps_cap=8, outputs=None):
    """The conventional PyTorch path on the same GPU and inputs: a cache that
    grows by ``torch.cat`` at every step (an O(t) copy instead of an
    O(d_k+d_v) append) and GQA by ``repeat_interleave`` of the KV heads (h_q
    copies of each KV row materialised and read instead of h_kv), then
    scores, softmax and the weighted sum as separate fp32 tensor operations.
    Sequences are handled one by one (their caches have different lengths).
    Returns timing and a byte model; the inputs are this workload's own."""
    import numpy as np
    import torch

    G = s.h_q // s.h_kv
    scale = float(s.scale32())
    # multi-step workloads: step 0 warms up, steps 1.. are timed (at most
    # steps_cap of them); a single decode is repeated on the same cache
    total = min(s.steps, steps_cap + 1) if s.steps else 1
    warm = 1 if total > 1 or not s.steps else 0
    timed = list(range(warm, total)) if s.steps else [0]
    Kb = [torch.from_numpy(np.ascontiguousarray(inp.K[b, :, :int(inp.lens[b])])).to(dev)
          for b in range(s.B)]
    Vb = [torch.from_numpy(np.ascontiguousarray(inp.V[b, :, :int(inp.lens[b])])).to(dev)
          for b in range(s.B)]
    if s.steps:
        kn = torch.from_numpy(inp.k_new[:total]).to(dev)
        vn = torch.from_numpy(inp.v_new[:total]).to(dev)
        qs = torch.from_numpy(inp.q_step[:total]).to(dev)
    else:
        qs = torch.from_numpy(inp.q[None]).to(dev)
    out = torch.empty((s.B, s.h_q, s.d_v), dtype=torch.float32, device=dev)

    def one_step(t):
        for b in range(s.B):
            if s.steps:
                Kb[b] = torch.cat([Kb[b], kn[t, b][:, None, :]], dim=1)
                Vb[b] = torch.cat([Vb[b], vn[t, b][:, None, :]], dim=1)
            Kx = Kb[b].repeat_interleave(G, dim=0) if G > 1 else Kb[b]   # [h_q, n, d_k]
            Vx = Vb[b].repeat_interleave(G, dim=0) if G > 1 else Vb[b]
            sc = torch.matmul(Kx, qs[t, b][:, :, None])[..., 0] * scale  # [h_q, n]
            a = torch.softmax(sc, dim=-1)
            out[b] = torch.matmul(a[:, None, :].contiguous(), Vx)[:, 0]

    if warm:
        one_step(0)                               # warm-up (allocator, kernels)
        torch.cuda.synchronize()
        if outputs is not None:                   # for the parity test
            outputs.append(out.double().cpu().numpy())
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record()
    for t in timed:
        one_step(t)
        if outputs is not None:
            torch.cuda.synchronize()
            outputs.append(out.double().cpu().numpy())
    t1.record()
    torch.cuda.synchronize()
    us = t0.elapsed_time(t1) * 1e3 / len(timed)
    lens = [int(Kb[b].shape[1]) for b in range(s.B)]
    F32 = 4
    d = s.d_k + s.d_v
    kv = sum(s.h_kv * n * d * F32 for n in lens)
    cat = 2 * kv if s.steps else 0                 # read the old cache, write the new one
    rep = (kv + G * kv) if G > 1 else 0           # read h_kv rows, write h_q copies
    attn = G * kv + s.B * s.h_q * d * F32         # read h_q rows per head, q, out
    return {
        "us_per_step": round(us, 2),
        "steps_timed": len(timed),
        "this_path_us_per_step": round(our_us_per_step, 2),
        "speedup_of_this_path": round(us / our_us_per_step, 2),
        "append": "torch.cat (the cache grows by a full copy each step)" if s.steps else None,
        "gqa": f"repeat_interleave x{G}" if G > 1 else None,
        "hbm_bytes_model_per_step": int(cat + rep + attn),
        "this_path_hbm_bytes_per_step": int(kv + s.B * s.h_q * d * F32 +
                                            (s.B * s.h_kv * d * F32 if s.steps else 0)),
        "final_len": lens,
    }


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=64)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="c5")
    ap.add_argument("--shape", default="",
                    help="a custom workload instead of --workload, e.g. "
                         "'B=8,h_q=32,h_kv=8,d_k=64,d_v=64,n_max=32768,steps=8' "
                         "(also len_lo, len_hi, rows; lengths default to n_max, less "
                         "steps*rows when there are steps)")
    ap.add_argument("--chunk-rows", type=int, default=0)
    ap.add_argument("--settle-seconds", type=float, default=0.3,
                    help="untimed repetitions of the step before the warm-up, so that "
                         "the GPU runs at its steady clock (0: none)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="budget of the CPU-oracle sample (0: skip)")
    ap.add_argument("--conventional", action="store_true",
                    help="also time the conventional PyTorch path (torch.cat cache, "
                         "repeat_interleave GQA) on the same inputs")
    ap.add_argument("--graph", action="store_true",
                    help="capture the timed steps in one HIP graph and replay it")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="only run a plain device copy of this size (for counter scaling)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py: this benchmark runs on one GPU; --gpus {args.gpus} is not "
              "supported (the decode would shard by KV head, each GPU holding whole "
              "query-head groups, with no exchange between GPUs)", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    from paper_2607_19456_amd import binding, traffic, workloads

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    if args.copy_calibration_mib:
        n = args.copy_calibration_mib << 20
        a = torch.empty(n // 4, dtype=torch.float32, device=dev).fill_(1.0)
        b = torch.empty_like(a)
        for _ in range(5):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": n, "launches": 5}))
        return 0

    shape = custom_shape(args.shape) if args.shape else workloads.get(args.workload)
    s = shape
    log(f"workload {s.name}: drawing inputs")
    t0 = time.perf_counter()
    inp = workloads.make(shape, seed=0, pad=0.0)
    log(f"inputs drawn in {time.perf_counter() - t0:.1f} s; copying to HBM")

    dK = torch.from_numpy(inp.K).to(dev)
    dV = torch.from_numpy(inp.V).to(dev)
    lens0 = torch.from_numpy(inp.lens).to(dev)
    dl = lens0.clone()
    nsteps_in = max(1, s.steps)
    if s.steps:
        dkn = torch.from_numpy(inp.k_new).to(dev)
        dvn = torch.from_numpy(inp.v_new).to(dev)
        dq = torch.from_numpy(inp.q_step).to(dev)
    else:
        dq = torch.from_numpy(inp.q[None]).to(dev)
    multi = s.rows > 1
    # A single decode whose slabs are each one chunk runs in the direct form
    # (one launch writes the output): time da_decode_attn as a whole then.
    out = torch.empty((s.B, s.h_q) + ((s.rows,) if multi else ()) + (s.d_v,),
                      dtype=torch.float32, device=dev)
    # The library's own segment size unless --chunk-rows asks for another
    # (then the tuning calls run; `chunk` is reported either way).
    ck = args.chunk_rows
    chunk = ck or binding.chunk_rows(s.B, s.h_q * s.rows, s.h_kv, s.n_max, s.d_k, s.d_v)
    direct = not s.steps and not multi and chunk >= s.n_max
    # A fused step on single-chunk slabs with one column block and
    # d_k + d_v <= 256 is one launch as well (da_decode_step, direct form).
    direct_step = (bool(s.steps) and not multi and not ck and chunk >= s.n_max
                   and s.h_q // s.h_kv <= 16 and s.d_k + s.d_v <= 256)
    if multi:
        ws = binding.alloc_multi_workspace(dq[0], dK, dV, ck)
    else:
        ws = binding.alloc_workspace(dq[0], dK, dV, ck)
    scale = float(s.scale32())
    stream = torch.cuda.current_stream()
    torch.cuda.synchronize()

    def step(i, ev_a=None, ev_b=None, ev_c=None):
        # One step: the append fused into the decode's partial kernel, then
        # the merge (which also advances len) -- da_decode_step, with the
        # partial kernel bracketed by events.
        t = i % nsteps_in
        st = torch.cuda.current_stream()   # the capture stream inside a graph
        if s.steps and t == 0 and i > 0:
            dl.copy_(lens0)              # a new pass over the multi-step sequence
        if ev_a is not None:
            ev_a.record(st)
        if multi:
            # several positions per step: da_decode_multi_step, both launches
            # inside the events
            binding.decode_multi_step(dq[t], dK, dV, dkn[t], dvn[t], dl, scale, out=out,
                                      workspace=ws, chunk_rows=ck, stream=st)
            if ev_b is not None:
                ev_b.record(st)
            return
        if direct:
            binding.decode_attn(dq[t], dK, dV, dl, scale, out=out, workspace=ws,
                                chunk_rows=ck, stream=st)
            if ev_b is not None:
                ev_b.record(st)
            return
        if direct_step:
            binding.decode_step(dq[t], dK, dV, dkn[t], dvn[t], dl, scale, out=out,
                                workspace=ws, stream=st)
            if ev_b is not None:
                ev_b.record(st)
            return
        if s.steps:
            binding.decode_partial(dq[t], dK, dV, dl, scale, ws, ck,
                                   k_new=dkn[t], v_new=dvn[t], stream=st)
        else:
            binding.decode_partial(dq[t], dK, dV, dl, scale, ws, ck, stream=st)
        if ev_b is not None:
            ev_b.record(st)
        binding.decode_merge(out, ws, s.B, s.h_q, s.h_kv, s.n_max, s.d_k, s.d_v,
                             ck, lens=dl if s.steps else None, stream=st)
        if ev_c is not None:
            ev_c.record(st)

    # The GPU comes out of the idle input-drawing phase at a low clock and
    # needs some tens of milliseconds of load to reach its steady clock (the
    # first ~10 ms batch of a 64-step run measured 6 % slower than the ones
    # after it).  Steady-state decoding keeps the GPU busy, so the step is
    # first repeated, untimed, for --settle-seconds of wall time; then come
    # the W warm-up steps and the K timed steps.
    settled = 0
    if args.settle_seconds > 0:
        t_settle = time.perf_counter()
        while time.perf_counter() - t_settle < args.settle_seconds:
            for _ in range(8):
                step(settled)
                settled += 1
            torch.cuda.synchronize()
        dl.copy_(lens0)
        log(f"settled the clock with {settled} untimed step(s)")
    log(f"warmup {args.warmup} step(s), chunk_rows={chunk}")
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    dl.copy_(lens0)
    torch.cuda.synchronize()

    # Host-side mirror of the lengths each timed step decodes over.
    lens_host = inp.lens.astype(np.int64)
    step_lens = []
    for i in range(args.steps):
        t = i % nsteps_in
        if s.steps:
            if t == 0 and i > 0:
                lens_host = inp.lens.astype(np.int64)
            lens_host = np.minimum(lens_host + s.rows, s.n_max)
        step_lens.append(lens_host.copy())

    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    if args.graph:
        # The timed steps as one graph (the graph holds no memset, and the
        # workspace counters come back to zero after each step), replayed once
        # from the same initial state.
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for i in range(args.steps):
                step(i)
        dl.copy_(lens0)
        torch.cuda.synchronize()
        stream = torch.cuda.current_stream()
        if args.settle_seconds > 0:
            # The capture leaves the GPU idle: one untimed replay brings the
            # clock back before the timed one.
            graph.replay()
            torch.cuda.synchronize()
            dl.copy_(lens0)
            torch.cuda.synchronize()
        log(f"timing {args.steps} step(s) as one graph replay")
        wall0 = time.perf_counter()
        start.record(stream)
        graph.replay()
        end.record(stream)
        torch.cuda.synchronize()
    else:
        # The K steps back to back, with nothing but their own launches on
        # the stream between the two events.
        log(f"timing {args.steps} step(s)")
        torch.cuda.synchronize()
        wall0 = time.perf_counter()
        start.record(stream)
        for i in range(args.steps):
            step(i)
        end.record(stream)
        torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    total_ms = start.elapsed_time(end)

    # Per-launch durations for the roofline: the same K steps once more, from
    # the same initial state, each launch bracketed by events.  They stay out
    # of the timed region above because every event recorded between two
    # launches holds the next one back (about 3 us each; three per step made
    # a long-context step ~10 us longer).
    dl.copy_(lens0)
    torch.cuda.synchronize()
    ev_a = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ev_b = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ev_c = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    for i in range(args.steps):
        step(i, ev_a[i], ev_b[i], ev_c[i])
    torch.cuda.synchronize()
    launch_ms = [a.elapsed_time(b) for a, b in zip(ev_a, ev_b)]
    merge_ms = None
    if not (multi or direct or direct_step):
        merge_ms = [b.elapsed_time(c) for b, c in zip(ev_b, ev_c)]
    log(f"per-launch pass: {sum(launch_ms) / len(launch_ms) * 1e3:.1f} us per "
        + ("step" if (multi or direct or direct_step) else "partial launch"))

    def step_bytes(lens, with_append=True):
        b = traffic.batch_decode_bytes(lens, s.h_q, s.h_kv, s.d_k, s.d_v, s.rows)
        if with_append:
            b += traffic.batch_append_bytes(s.B, s.h_kv, s.d_k, s.d_v, s.rows)
        return b

    alg_bytes = sum(step_bytes(l, bool(s.steps)) for l in step_lens)
    # The partial kernel of a step also writes the appended rows (Prop. 2).
    append_b = traffic.batch_append_bytes(s.B, s.h_kv, s.d_k, s.d_v, s.rows) if s.steps else 0
    if multi or direct or direct_step:   # the events hold the whole step
        launch_bytes = [step_bytes(l, bool(s.steps)) for l in step_lens]
    else:
        launch_bytes = [traffic.batch_partial_bytes(l, s.h_q, s.h_kv, s.d_k, s.d_v) + append_b
                        for l in step_lens]
    ms_per_step = total_ms / args.steps
    value = alg_bytes / (total_ms * 1e-3) / 1e9
    launch_avg_ms = sum(launch_ms) / len(launch_ms)
    achieved = (sum(launch_bytes) / len(launch_bytes)) / (launch_avg_ms * 1e-3) / 1e9

    result = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": s.name,
            "B": s.B, "h_q": s.h_q, "h_kv": s.h_kv, "d_k": s.d_k, "d_v": s.d_v,
            "n_max": s.n_max,
            "initial_len": [int(x) for x in inp.lens],
            "steps_per_sequence": s.steps,
            "rows_per_step": s.rows,
            "chunk_rows": chunk,
            "step": ("da_decode_multi_step (T-row append fused, causal T-row decode)"
                     if multi else
                     "da_decode_attn (direct form: one launch, no merge)" if direct else
                     "da_decode_step (direct form: append, decode and len advance in one "
                     "launch)" if direct_step else
                     "decode_partial with fused kv_append + decode_merge" if s.steps
                     else "decode_partial + decode_merge"),
            "graph": bool(args.graph),
        },
        "settle_steps_untimed": settled,
        "us_per_step": round(ms_per_step * 1e3, 2),
        "step_timing": ("one graph replay of the K steps between two events" if args.graph
                        else "two events around the K steps, none between them"),
        "hbm_roofline_frac_step": round(value / HBM_PEAK_GBPS, 4),
        "algorithmic_bytes_per_step": int(alg_bytes / args.steps),
        "host_wall_s": round(wall, 4),
        "roofline": {
            "bound": "hbm",
            "kernel": ("decode_partial_kernel + decode_merge_kernel (the whole step)"
                       if multi else
                       "decode_partial_kernel (direct form, the whole decode)" if direct
                       else "decode_partial_kernel (direct form, the whole step)" if direct_step
                       else "decode_partial_kernel"),
            "achieved": round(achieved, 2),
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBPS, 4),
            "traffic": None if multi else counter_traffic(s.name),
            "avg_launch_us": round(launch_avg_ms * 1e3, 2),
            "timing": ("HIP events around each step" if multi or direct or direct_step
                       else "HIP events around each partial launch")
                      + ", in a second pass over the same K steps (the timed region has "
                        "no events between its launches)",
            "algorithmic_bytes_per_launch": int(sum(launch_bytes) / len(launch_bytes)),
        },
    }
    log(f"{ms_per_step * 1e3:.1f} us/step, {value:.0f} GB/s; partial "
        f"{launch_avg_ms * 1e3:.1f} us at {achieved:.0f} GB/s")

    # The parts of a step, each timed with events on the same stream: the
    # partial kernel (with the fused append) and the merge of the timed
    # steps above, then the standalone append (da_kv_append, or
    # da_kv_append_rows for several rows per step) over the same steps on
    # its own.
    comps = {"decode_partial_us": None, "decode_merge_us": None,
             "kv_append_standalone_us": None, "kv_append_bytes_per_step": None}
    if merge_ms is not None:
        comps["decode_partial_us"] = round(launch_avg_ms * 1e3, 2)
        comps["decode_merge_us"] = round(sum(merge_ms) / len(merge_ms) * 1e3, 2)
    if s.steps:
        dl.copy_(lens0)
        torch.cuda.synchronize()
        ea = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
        eb = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
        for i in range(args.steps):
            t = i % nsteps_in
            if t == 0 and i > 0:
                dl.copy_(lens0)
            ea[i].record(stream)
            if multi:
                binding.kv_append_rows(dK, dV, dkn[t], dvn[t], dl, stream=stream)
            else:
                binding.kv_append(dK, dV, dkn[t], dvn[t], dl, stream=stream)
            eb[i].record(stream)
        torch.cuda.synchronize()
        comps["kv_append_standalone_us"] = round(
            sum(a.elapsed_time(b) for a, b in zip(ea, eb)) / args.steps * 1e3, 2)
        comps["kv_append_bytes_per_step"] = traffic.batch_append_bytes(
            s.B, s.h_kv, s.d_k, s.d_v, s.rows)
        dl.copy_(lens0)
        log(f"standalone append: {comps['kv_append_standalone_us']} us per step")
    result["step_components"] = comps

    # The machine's practical read ceiling on the same K and V allocations:
    # a plain non-temporal streaming read of every byte (not the decode).
    ceil_gbps, ceil_bytes = read_ceiling(dK, dV, stream)
    result["roofline"]["ceiling"] = {
        "achieved": round(ceil_gbps, 2), "unit": "GB/s", "bytes": ceil_bytes,
        "kind": "streaming read of the same K and V allocations (hbm_probe: 16-byte "
                "non-temporal loads, 8 in flight per thread, one workgroup per CU), "
                "mean of 5 after 1 warm-up",
        "frac": round(achieved / ceil_gbps, 4),
    }
    log(f"read ceiling on the same buffers: {ceil_gbps:.0f} GB/s; the decode's partial "
        f"kernel reaches {achieved / ceil_gbps:.1%} of it")

    first_out = None
    if args.cpu_seconds > 0:
        # The first step once more from the initial lengths (it rewrites its
        # appended rows with the same values), for the oracle check below.
        dl.copy_(lens0)
        step(0)
        torch.cuda.synchronize()
        first_out = out.double().cpu().numpy()
    del dK, dV
    torch.cuda.empty_cache()
    if args.conventional:
        if s.rows > 1:
            result["conventional"] = None
        else:
            log("conventional PyTorch path on the same inputs")
            result["conventional"] = conventional_leg(s, inp, dev, ms_per_step * 1e3)
            log(f"conventional: {result['conventional']['us_per_step']} us/step")
            torch.cuda.empty_cache()
    if args.cpu_seconds > 0:
        log("cpu_baseline: timing the oracle on this host")
        # the oracle replays the workload from its initial state
        result["cpu_baseline"] = cpu_baseline(inp, args.cpu_seconds, step_bytes, first_out)
        result["max_abs_err_vs_oracle"] = result["cpu_baseline"]["max_abs_err_first_step"]
        if s.name in ("mha1_d64_n128", "gqa32x8_b16_d128_n8192"):
            # the small and the GQA-4 single decode also on one thread
            log("cpu_baseline: the oracle on one thread")
            one = cpu_baseline(inp, min(args.cpu_seconds, 10.0), step_bytes, None, threads=1)
            result["cpu_baseline"]["one_thread"] = {
                k: one[k] for k in ("value", "unit", "cores", "sample", "seconds_per_step")}
        log(f"max-abs-err of the first step vs the oracle: {result['max_abs_err_vs_oracle']:.3e}")
    else:
        result["cpu_baseline"] = None
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
