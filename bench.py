#!/usr/bin/env python
"""Benchmark of one retrospective sparse-attention decode step per layer on one GPU.

Workload (default): a Llama-3-8B-shaped attention layer, batch 1, 8 KV heads,
32 query heads, head_dim 128, bf16, 32K-token context in pages of 16, token
budget 2048 (128 pages), retrospective window W = 16 past queries.  Seeded
synthetic keys / values / queries (no dataset or weights are needed).

A "step" is one whole decode step (append, page scoring, top-k + mask,
attention over the W+1 window queries, merge into the output cache) for each of
--layers independent layer replicas: with 32 replicas (an 8B model's layer
count) the data touched per step is far above the 256 MB Infinity Cache, so the
bytes really come from HBM.  Steps are captured as HIP graphs (one per step) and
replayed back to back in the timed region.

Prints one JSON line with the throughput (effective HBM GB/s of the whole step,
algorithmic bytes / time), microseconds per layer per step, the roofline of the
dominant kernel (where retro_step is one launch, that launch: the whole step;
else its scores + selection + attention launch, timed alone with HIP events),
the gather phase alone (the attention kernel over the step's selection, timed
with HIP events) and the CPU oracle's rate on a bounded sample.
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

METRIC = "retro_step µs/layer/decode-step + effective HBM GB/s (% peak), 32K ctx B=2048 W=16"
PEAK_HBM_GBS = 8000.0
STEP_SRC = [os.path.join(ROOT, "paper_2508_09001_amd", "csrc", f)
            for f in ("step_attend.hip", "roles.h", "threshold.h", "internal.h")]
COUNTERS = os.path.join(ROOT, "profiles", "step_attend_kernel_llama3-8b-32k_counters.json")


def _args():
    p = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=16, help="timed decode steps")
    p.add_argument("--warmup", type=int, default=4, help="untimed decode steps")
    p.add_argument("--layers", type=int, default=32, help="layer replicas rotated per step")
    p.add_argument("--config", type=int, default=1, help="workload index (1 = headline)")
    p.add_argument("--window", type=int, default=None,
                   help="override the workload's window W (W = 0: no retrospection)")
    p.add_argument("--budget", type=int, default=None,
                   help="override the workload's token budget B")
    p.add_argument("--reuse-interval", type=int, default=None,
                   help="top-k selection reuse: refresh the selection every f steps (f >= 2)")
    p.add_argument("--budget-permille", type=int, default=None,
                   help="relative budget in thousandths of the context (0: fixed budget)")
    p.add_argument("--update-kv", action="store_true",
                   help="UpdateKV of the window's W past tokens before every step (Alg. 1)")
    p.add_argument("--attend-reps", type=int, default=4,
                   help="scores + selection + attention launches per layer in the roofline measurement")
    p.add_argument("--cpu-seconds", type=float, default=15.0,
                   help="budget of the CPU oracle sample (0 skips it)")
    p.add_argument("--decoder", type=int, default=0,
                   help="instead: a stack of this many layers with projections and "
                        "re-embedding, timed per token at each --decoder-windows value")
    p.add_argument("--decoder-windows", default="0,2,4,8,16",
                   help="windows W compared in --decoder mode")
    p.add_argument("--decoder-batch", type=int, default=None,
                   help="in --decoder mode, sequences decoded together (all at the workload's "
                        "first context length)")
    p.add_argument("--decoder-torch-proj", action="store_true",
                   help="in --decoder mode, run the projections on torch.matmul instead")
    p.add_argument("--calib-copy", action="store_true",
                   help="only run a 512 MiB device copy (counter calibration) and exit")
    return p.parse_args()


def _sha(paths):
    h = hashlib.sha256()
    for p in paths:
        with open(p, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def _step_path(launches, reuse=0):
    """The launch sequence retro_step takes (the library's own choice, no flags)."""
    if launches == 1:
        path = "one launch: scores, selection, attention, combine + merge"
    else:
        path = (f"{launches} launches: scores (+ selection), [selection +] attention, "
                "combine + merge")
    if reuse >= 2:
        path = (f"refresh steps (t mod {reuse} == 0): {path}; other steps keep the selection: "
                "4 launches: append, mask, attention, combine + merge")
    return path


def algorithmic_bytes(spec, seq_lens, num_selected):
    """Bytes one layer-step must move at minimum (per the step's definition)."""
    elt = 2 if spec.dtype == "bf16" else 4
    b, hk, hq, d, P, W = spec.batch, spec.num_kv_heads, spec.num_q_heads, spec.head_dim, \
        spec.page_size, spec.window
    n_pages = sum(-(-int(L) // P) for L in seq_lens)
    k_sum = int(sum(int(x) for x in num_selected.reshape(-1)))     # over (b, h)
    # with top-k reuse (refresh every f steps) only the refresh steps scan the
    # digests and select: their bytes averaged over the steps
    f = spec.reuse_interval if spec.reuse_interval >= 2 else 1
    digest = n_pages * hk * 2 * d * elt // f
    gather = k_sum * P * 2 * d * elt
    queries = b * (W + 1) * hq * d * elt
    ring = 2 * b * W * hq * (d + 1) * 4
    out = b * (W + 1) * hq * (d + 1) * 4
    mask = 12 * k_sum
    append = spec.tokens_per_step * (b * hk * d * elt * 2 + b * hk * 2 * d * elt * 2)
    # what the selection reads besides the scores: last_loaded per (b, h), the page table per b
    select_reads = (n_pages * hk * 4 + n_pages * 4) // f
    return dict(total=digest + gather + queries + ring + out + mask + append, digest=digest,
                gather=gather, queries=queries, ring=ring, out=out, mask=mask, append=append,
                select_reads=select_reads)


def _calib_copy():
    """A plain elementwise kernel that reads n bytes and writes n bytes: the
    reference for scaling the FETCH_SIZE / WRITE_SIZE counters to bytes."""
    import torch
    n = 512 << 20
    src = torch.ones(n // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        torch.neg(src, out=dst)
    torch.cuda.synchronize()
    print(json.dumps({"calib_copy_bytes": n, "launches": 3}))


def main():
    args = _args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the step shards "
              "by KV head or sequence with no communication, see the design notes", file=sys.stderr)
        sys.exit(2)
    from paper_2508_09001_amd import binding
    if not os.path.exists(binding.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    import numpy as np
    import torch

    import workloads as W
    from paper_2508_09001_amd.layer import RetroLayer

    if args.calib_copy:
        _calib_copy()
        return
    if args.decoder > 0:
        decoder_bench(args)
        return
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    base_spec = W.config(args.config)
    if args.window is not None:
        base_spec = base_spec.replace(window=args.window)
    if args.budget is not None:
        base_spec = base_spec.replace(budget=args.budget)
    if args.budget_permille is not None:
        base_spec = base_spec.replace(budget_permille=args.budget_permille)
    if args.reuse_interval is not None:
        base_spec = base_spec.replace(reuse_interval=args.reuse_interval)
    need = args.warmup + 2 * args.steps
    spec = base_spec if need <= base_spec.steps else base_spec.replace(steps=need)
    L = args.layers

    # ---- inputs: prefill + per-step tokens and query windows, resident on the GPU
    gen = W.Generator(spec)
    pre = gen.prefill()
    qw = W.QueryWindow(spec)
    steps_in = []
    for t in range(need):
        k_new, v_new, q = gen.step(t)
        win = qw.push(q).copy()
        steps_in.append(tuple(torch.from_numpy(np.ascontiguousarray(x)).to(
            "cuda", dtype=torch.bfloat16 if spec.dtype == "bf16" else torch.float32)
            for x in (win, k_new, v_new)))
    layers = [RetroLayer.for_spec(spec) for _ in range(L)]
    for b, (k, v) in enumerate(pre):
        layers[0].prefill(b, k, v)
    for lay in layers[1:]:
        for name in ("k_cache", "v_cache", "digest", "seq_lens", "last_loaded"):
            getattr(lay, name).copy_(getattr(layers[0], name))
        lay._lens = list(layers[0]._lens)
    torch.cuda.synchronize()

    # UpdateKV inputs: seeded synthetic re-embedded keys / values of the W past
    # tokens, resident on the device like the step's other inputs
    upd = None
    if args.update_kv and spec.window > 0:
        gen_u = torch.Generator().manual_seed(7)
        td = torch.bfloat16 if spec.dtype == "bf16" else torch.float32
        shape = (spec.batch, spec.window, spec.num_kv_heads, spec.head_dim)
        upd = [tuple(torch.randn(shape, generator=gen_u).to("cuda", dtype=td) for _ in range(2))
               for _ in range(4)]

    def run_step(t):
        win, k_new, v_new = steps_in[t]
        for lay in layers:
            if upd is not None and t > 0:
                lay.update_kv(*upd[t % len(upd)])
            if k_new.shape[0] > 1:  # the step's tokens before its last, in one launch
                lay.append_tokens(t, k_new[:-1], v_new[:-1])
            lay.step(t, win, k_new[-1], v_new[-1])

    for t in range(args.warmup):
        run_step(t)
    torch.cuda.synchronize()

    # ---- timed region: K steps replayed from HIP graphs
    t0 = args.warmup
    graphs = []
    for t in range(t0, t0 + args.steps):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            run_step(t)
        graphs.append(g)
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record()
    for g in graphs:
        g.replay()
    ev1.record()
    torch.cuda.synchronize()
    ms_graph = ev0.elapsed_time(ev1)
    seq_mid = layers[0].seq_lens.cpu().numpy()
    nsel = layers[0].num_selected.cpu().numpy()

    # ---- eager launches of the next K steps, for comparison
    t1 = t0 + args.steps
    ev0.record()
    for t in range(t1, t1 + args.steps):
        run_step(t)
    ev1.record()
    torch.cuda.synchronize()
    ms_eager = ev0.elapsed_time(ev1)

    def graph_us(fn):
        """HIP-event time per launch of a graph of L * attend_reps launches of fn."""
        gr = torch.cuda.CUDAGraph()
        with torch.cuda.graph(gr):
            for _ in range(args.attend_reps):
                for lay in layers:
                    fn(lay)
        torch.cuda.synchronize()
        ev0.record()
        gr.replay()
        ev1.record()
        torch.cuda.synchronize()
        return ev0.elapsed_time(ev1) * 1000.0 / (args.attend_reps * L)

    from paper_2508_09001_amd import binding as B
    launches = B.retro_step_launches(layers[0].dims)
    nbytes = algorithmic_bytes(spec, seq_mid, nsel)
    us_layer_step = ms_graph * 1000.0 / (args.steps * L)
    gbs = nbytes["total"] / (us_layer_step * 1e-6) / 1e9
    last = t1 + args.steps - 1
    win_last = steps_in[last][0]
    n_att = args.attend_reps * L
    traffic = None
    if launches == 1 and spec.reuse_interval < 2:
        # the dominant kernel is the step itself: its launches in the timed
        # graphs (one per layer-step), every algorithmic byte of the step
        kernel, us_kernel, kernel_bytes, n_kernel = ("step_attend_kernel", us_layer_step,
                                                     nbytes["total"], args.steps * L)
        if os.path.exists(COUNTERS):
            with open(COUNTERS) as f:
                cnt = json.load(f)
            if cnt.get("source_sha256") == _sha(STEP_SRC):
                traffic = cnt.get("hbm_bytes_per_launch")
    else:
        # the step's scores + selection + attention launch alone: digests ->
        # scores -> selection -> gather, queries
        kernel = "scores + selection + attention launch"
        us_kernel = graph_us(lambda lay: lay.step_attend_partials(last, win_last))
        kernel_bytes = (nbytes["digest"] + nbytes["gather"] + nbytes["queries"] +
                        nbytes["select_reads"])
        n_kernel = n_att
    kernel_gbs = kernel_bytes / (us_kernel * 1e-6) / 1e9
    # the gather phase alone: the attention kernel over the step's selection
    # (the pages' keys and values, the window's queries, the selection rows)
    us_gather = graph_us(lambda lay: lay.attend_partials(last, win_last))
    gather_bytes = nbytes["gather"] + nbytes["queries"] + nbytes["mask"]
    gather_gbs = gather_bytes / (us_gather * 1e-6) / 1e9

    result = {
        "metric": METRIC,
        "value": round(gbs, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_graph / args.steps, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": spec.dtype,
        "data": "synthetic",
        "config": {"workload": spec.name, "batch": spec.batch, "kv_heads": spec.num_kv_heads,
                   "q_heads": spec.num_q_heads, "head_dim": spec.head_dim,
                   "context": int(spec.prefill[0]), "page_size": spec.page_size,
                   "budget_tokens": spec.budget, "budget_permille": spec.budget_permille,
                   "window": spec.window, "update_kv": bool(upd is not None),
                   "reuse_interval": spec.reuse_interval,
                   "layers_rotated": L,
                   "launch": "hip-graph per step",
                   "step_path": _step_path(launches, spec.reuse_interval)},
        "us_per_layer_step": round(us_layer_step, 3),
        "us_per_layer_step_eager": round(ms_eager * 1000.0 / (args.steps * L), 3),
        "frac_of_peak_hbm": round(gbs / PEAK_HBM_GBS, 4),
        "bytes_per_layer_step": nbytes,
        "roofline": {"bound": "hbm", "kernel": kernel,
                     "achieved": round(kernel_gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": round(kernel_gbs / PEAK_HBM_GBS, 4), "traffic": traffic,
                     "bytes_per_launch": kernel_bytes, "us_per_launch": round(us_kernel, 3),
                     "launches": n_kernel},
        "gather_phase": {"kernel": "attend_kernel (retro_decode_attend_partials)",
                         "bytes_per_launch": gather_bytes, "us_per_launch": round(us_gather, 3),
                         "achieved": round(gather_gbs, 1), "unit": "GB/s",
                         "frac": round(gather_gbs / PEAK_HBM_GBS, 4), "launches": n_att},
    }

    if args.cpu_seconds > 0:
        result["cpu_baseline"] = cpu_baseline(spec, pre, args.cpu_seconds)
    print(json.dumps(result), flush=True)


def decoder_bench(args):
    """Per-token latency of a stack of args.decoder layers (random-weight query, key,
    value and output projections around each layer's step; the past rows re-embedded
    and their keys and values overwritten), at every window in --decoder-windows:
    the analogue of the paper's throughput-versus-window table.  Inputs are drawn on
    the device from seeded generators; each timed step is replayed from its own HIP
    graph."""
    import torch

    import workloads as W
    from paper_2508_09001_amd.decode import RetroDecoder, layer_kwargs

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    base = W.config(args.config)
    if args.budget_permille is not None:
        base = base.replace(budget_permille=args.budget_permille)
    if args.decoder_batch is not None:
        base = base.replace(batch=args.decoder_batch,
                            prefill=(base.prefill[0],) * args.decoder_batch)
    windows = [int(x) for x in args.decoder_windows.split(",")]
    L = args.decoder
    warmup = max(args.warmup, max(windows) + 1)   # every past row re-embedded from then on
    need = warmup + args.steps + 1
    spec0 = base.replace(steps=max(base.steps, need))
    dev = torch.device("cuda")
    td = torch.bfloat16 if spec0.dtype == "bf16" else torch.float32
    dm = spec0.num_q_heads * spec0.head_dim
    g = torch.Generator(device=dev).manual_seed(2508)

    def randn(*shape, scale=1.0):
        return (torch.randn(*shape, generator=g, device=dev) * scale).to(td)

    hq_d, hk_d = spec0.num_q_heads * spec0.head_dim, spec0.num_kv_heads * spec0.head_dim
    weights = [dict(wq=randn(dm, hq_d, scale=dm ** -0.5), wk=randn(dm, hk_d, scale=dm ** -0.5),
                    wv=randn(dm, hk_d, scale=dm ** -0.5),
                    wo=randn(hq_d, dm, scale=(hq_d * L) ** -0.5)) for _ in range(L)]
    prompts = [[(randn(n, spec0.num_kv_heads, spec0.head_dim),
                 randn(n, spec0.num_kv_heads, spec0.head_dim)) for n in spec0.prefill]
               for _ in range(L)]
    emb = randn(spec0.batch, need + max(windows), dm)
    ms, lib_proj = {}, {}
    for w in windows:
        spec = spec0.replace(window=w)
        dec = RetroDecoder(weights, library_projections=not args.decoder_torch_proj,
                           **layer_kwargs(spec))
        for layer in range(L):
            for b, (k, v) in enumerate(prompts[layer]):
                dec.prefill(layer, b, k, v)
        off = max(windows)
        wins = [emb[:, off + t - w:off + t + 1].contiguous() for t in range(need)]
        for t in range(warmup):
            dec.step(t, wins[t])
        torch.cuda.synchronize()
        graphs = []
        for t in range(warmup, warmup + args.steps):
            gr = torch.cuda.CUDAGraph()
            with torch.cuda.graph(gr):
                dec.step(t, wins[t])
            graphs.append(gr)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for gr in graphs:
            gr.replay()
        e1.record()
        torch.cuda.synchronize()
        ms[w] = e0.elapsed_time(e1) / args.steps
        print(f"[decoder] W={w}: {ms[w]:.4f} ms/token over {L} layers, batch {spec.batch}, "
              f"projections {'library' if dec.fused else 'torch.matmul'}", file=sys.stderr,
              flush=True)
        lib_proj[w] = bool(dec.fused)
        del graphs, dec, wins
        torch.cuda.empty_cache()
    w_main = max(windows)
    base_ms = ms.get(0)
    result = {
        "metric": "decode_ms_per_token",
        "value": round(ms[w_main], 4),
        "unit": "ms/token",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": warmup,
        "ms_per_step": round(ms[w_main], 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": spec0.dtype,
        "data": "synthetic",
        "config": {"workload": f"{spec0.name} x {L} layers with projections",
                   "batch": spec0.batch, "context": int(spec0.prefill[0]), "layers": L,
                   "d_model": dm, "budget_tokens": spec0.budget,
                   "budget_permille": spec0.budget_permille, "window": w_main,
                   "launch": "hip-graph per token",
                   "projections": {str(w): "library" if v else "torch.matmul"
                                   for w, v in lib_proj.items()}},
        "ms_per_token_by_window": {str(w): round(v, 4) for w, v in ms.items()},
        "tokens_per_s_by_window": {str(w): round(spec0.batch * 1000.0 / v, 1)
                                   for w, v in ms.items()},
    }
    if base_ms:
        result["overhead_vs_w0_pct"] = {str(w): round(100.0 * (v / base_ms - 1.0), 2)
                                        for w, v in ms.items() if w != 0}
    print(json.dumps(result), flush=True)


def _cpu_model():
    """The host CPU's model name, as /proc/cpuinfo reports it."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cpu_baseline(spec, pre, budget_s):
    """The CPU oracle on the same workload: untimed ramp-up of the window, then
    decode steps of one layer until the time budget is used."""
    import numpy as np

    import oracle
    import workloads as W
    gen = W.Generator(spec)
    gen.prefill()          # regenerates the same prefill (keeps the generator's key store)
    orc = oracle.Oracle.for_spec(spec)
    for b, (k, v) in enumerate(pre):
        orc.prefill(b, k, v)
    qw = W.QueryWindow(spec)
    t = 0
    # the window's ramp-up, leaving at least a few steps to time
    ramp = min(spec.window, spec.steps - 4)
    for t in range(ramp):
        k_new, v_new, q = gen.step(t)
        orc.step(t, k_new, v_new, qw.push(q).copy())
    n, spent, last = 0, 0.0, None
    while (spent < budget_s or n == 0) and t + 1 < spec.steps:
        t += 1
        k_new, v_new, q = gen.step(t)
        win = qw.push(q).copy()
        s0 = time.perf_counter()
        last = orc.step(t, k_new, v_new, win)
        spent += time.perf_counter() - s0
        n += 1
    us = spent / max(n, 1) * 1e6
    nb = algorithmic_bytes(spec, orc.seq_lens, last["num_selected"])
    return {"value": round(nb["total"] / (us * 1e-6) / 1e9, 4), "unit": "GB/s",
            "us_per_layer_step": round(us, 1), "cores": oracle.num_threads(), "kind": "oracle",
            "cpu_model": _cpu_model(), "nproc": len(os.sched_getaffinity(0)),
            "omp_num_threads": os.environ.get("OMP_NUM_THREADS"),
            "sample": f"{n} decode steps of one layer of {spec.name} after {ramp} untimed "
                      f"steps (steps {ramp + 1}..{t}), fp64 attention, OpenMP"}


if __name__ == "__main__":
    main()
