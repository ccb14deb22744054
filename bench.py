"""Benchmark of the ReSA decode hot path on one MI355X.

A step is one decode token of one attention layer for the whole batch:
append the token's K/V (online block-summary update), select blocks (pooled
query, Quest score, top-n) and run block-sparse flash-decoding; every f-th
step of a layer also runs the dense rectification of its last f rows. By
default the step is resa_append_select then resa_sparse_decode (--mode two);
--mode step runs one launch of resa_decode_step, --mode three (--separate)
resa_append_kv, resa_select_blocks and resa_sparse_decode. The default
workload is the 64K batch-8 decode loop (32 query / 8 kv heads, head_dim 128,
block 16, sparsity 0.9 with a 2048-token minimum, f = 32, LogNormal(0, 0.5)
key channels). Steps cycle through `--layers` independent layer caches, as a
model's layers do, so data reused from one step to the next cannot be served
by the 256 MB last-level cache.

Prints one JSON line. `value` is the GPU time per step of the timed steps
(HIP events on the launch stream around the whole loop) with rectification
at its amortised rate of one call per f steps: the calls inside the timed
window are replaced by their measured per-call duration / f, and a window too
short to hold any (fewer than f steps per layer) gets one separately timed
call per layer, so short and long runs measure the same configured step
(`timed_gpu_us_per_step` is the raw timed figure). Every timed region starts
right after a few milliseconds of streaming reads (--burst-ms), so that it is
timed at the clocks of a loop running back to back rather than while they
ramp up after a host synchronisation. By default the timed steps are
recorded once into a HIP graph and replayed, as a serving loop would run
them; `--eager` launches every step from the host instead (the gaps between
host launches then count too). The per-kernel figures come from a second
pass that replays every launch of one kernel from the timed loop back to
back between two events. `roofline` is for the step's dominant kernel: the
fused step (bytes of the block summaries and of the selected K/V blocks) or,
with --mode two / three, the sparse decode (selected K/V); `decode_roofline`
is always the standalone sparse-decode kernel on the same selections;
`rectify_roofline` gives the rectification call's HBM fraction (every
group's K and V read once) and its matrix-core fraction (4 * 128 flops per
query head, window row and visible key); `stream_read_ceiling` is the read
bandwidth a plain streaming kernel reaches on the same GPU.
"""
from __future__ import annotations

import argparse
import ctypes as C
import hashlib
import json
import math
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
MFMA_PEAK_TFLOPS = 2500.0  # dense bf16 / fp16 matrix-core peak
METRIC = "sparse decode µs/step + achieved HBM GB/s (% roofline) at 64K/256K ctx"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=128)
    p.add_argument("--warmup", type=int, default=32)
    p.add_argument("--workload", default="long_64k",
                   choices=["long_64k", "extreme_256k", "qwen7b_32k", "tiny_4k", "sweep_64k"])
    p.add_argument("--layers", type=int, default=4)
    p.add_argument("--block-size", type=int, default=None)
    p.add_argument("--sparsity", type=float, default=None)
    p.add_argument("--rectify-every", type=int, default=None)
    p.add_argument("--dense", action="store_true", help="dense baseline: decode over every block")
    p.add_argument("--sweep", action="store_true",
                   help="64K batch-8 sweep: block size x sparsity x rectify interval, and dense decoding")
    p.add_argument("--breakdown", action="store_true",
                   help="latency breakdown at 16K/64K/256K (batch 8) against dense decoding")
    p.add_argument("--paged", action="store_true",
                   help="keep K and V in a shuffled page pool behind a block table")
    p.add_argument("--eager", dest="graph", action="store_false",
                   help="launch every timed step from the host instead of replaying them "
                        "from one HIP graph")
    p.add_argument("--prefill", action="store_true",
                   help="time prefill (chunked and whole-prompt) through the rectification call")
    p.add_argument("--mode", choices=["step", "two", "three"], default="two",
                   help="step: resa_decode_step (append + select + decode in one launch); "
                        "two: resa_append_select then resa_sparse_decode; three: resa_append_kv, "
                        "resa_select_blocks, resa_sparse_decode")
    p.add_argument("--separate", dest="mode", action="store_const", const="three",
                   help="same as --mode three")
    p.add_argument("--splits", type=int, default=0,
                   help="decode splits per (sequence, kv head); 0 = the library's choice")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-budget", type=float, default=20.0, help="seconds of oracle work")
    p.add_argument("--burst-ms", type=float, default=5.0,
                   help="GPU busy time (streaming reads) launched right before each timed region, "
                        "with no synchronisation in between")
    p.add_argument("--cap-pad", type=int, default=0,
                   help="extra cache capacity in tokens (layout experiments)")
    p.add_argument("--stream-probe", type=int, default=2 ** 31,
                   help="bytes of the stream-read ceiling measurement (0: skip)")
    p.add_argument("--copy-probe", type=int, default=0,
                   help="bytes of one plain device copy before the timed steps (counter reference)")
    return p.parse_args()


def workload_of(args):
    import workloads as W
    w = W.WORKLOADS[args.workload]
    kw = {}
    if args.block_size:
        kw["block_size"] = args.block_size
    if args.sparsity is not None:
        kw["sparsity"] = args.sparsity
    if args.rectify_every:
        kw["rectify_every"] = args.rectify_every
    return w.with_(**kw) if kw else w


def describe(w, layers, dense):
    return (f"{w.name}: batch {w.batch}, {w.num_q_heads} query / {w.num_kv_heads} kv heads, "
            f"head_dim {w.head_dim}, context {w.seq_len} growing by one token per step, "
            f"block {w.block_size}, " + ("dense (all blocks)" if dense else
                                          f"sparsity {w.sparsity} with a {w.min_tokens}-token minimum, ")
            + f"rectify every {w.rectify_every} steps, {layers} layer caches in rotation")


# The sources each timed kernel is compiled from (its own file and the
# headers holding its device code): a change to any of them retires the
# kernel's HBM counter figures.
KERNEL_SOURCES = {
    "k_decode": ["decode.hip", "decode_impl.h", "resa_device.h", "resa_internal.h"],
    "k_step": ["step.hip", "select_impl.h", "decode_impl.h", "resa_device.h", "resa_internal.h"],
}


def kernel_sources_sha256(kernel: str) -> str:
    """sha256 over the kernel's source files, in KERNEL_SOURCES order (each
    file's name, a NUL, its bytes)."""
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[kernel]:
        h.update(f.encode() + b"\0")
        with open(os.path.join(ROOT, "paper_2506_04108_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def traffic_from_profile(kernel: str, stem: str | None):
    """HBM bytes per launch measured by rocprofv3 PMC counters, read from
    profiles/<stem>_pmc.md (stem = kernel and workload, e.g.
    sparse_decode_long64k) if that profile was taken on the current kernel
    sources; else None (also for variants: dense, paged, overridden sizes)."""
    if stem is None:
        return None
    path = os.path.join(ROOT, "profiles", f"{stem}_pmc.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m = re.search(r"source_sha256:\s*([0-9a-f]{64})", text)
    t = re.search(r"traffic_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not m or not t:
        return None
    return float(t.group(1)) if m.group(1) == kernel_sources_sha256(kernel) else None


def cpu_baseline(w, budget_s):
    """The oracle timed on host cores on a bounded sample of the same workload."""
    import numpy as np
    import oracle as O
    import workloads as W
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        cores = 1
    groups = w.batch * w.num_kv_heads
    g = w.group_size
    f = w.rectify_every
    t_step = []
    t_rect = []
    t0 = time.perf_counter()
    sampled = 0
    for gi in range(groups):
        bi, hi = divmod(gi, w.num_kv_heads)
        k, v = W.group_kv(w, bi, hi)
        cap = w.seq_len + f + 1
        K = np.zeros((1, 1, cap, w.head_dim))
        V = np.zeros((1, 1, cap, w.head_dim))
        K[0, 0, :w.seq_len] = O.bf16_to_f64(k)
        V[0, 0, :w.seq_len] = O.bf16_to_f64(v)
        st = O.DecodeState(K, V, [w.seq_len], w.block_size)
        q = O.bf16_to_f64(W.decode_query(w, 0))[bi:bi + 1, hi * g:(hi + 1) * g]
        kn, vn = W.decode_kv(w, 0)
        a = time.perf_counter()
        st.append(O.bf16_to_f64(kn)[bi:bi + 1, hi:hi + 1], O.bf16_to_f64(vn)[bi:bi + 1, hi:hi + 1])
        _, idx, _ = st.select(q, w.sparsity, w.min_blocks, w.n_local)
        st.attend(q, idx, w.sm_scale)
        t_step.append(time.perf_counter() - a)
        if gi == 0:
            qf = np.random.default_rng(0).standard_normal((1, g, f, w.head_dim))
            kf = st.K[0:1, 0:1, st.L[0] - f:st.L[0]]
            a = time.perf_counter()
            st.rectify(qf, kf, st.V[0:1, 0:1, st.L[0] - f:st.L[0]], f, w.sm_scale)
            t_rect.append(time.perf_counter() - a)
        sampled += 1
        if time.perf_counter() - t0 > budget_s:
            break
    per_group_step = sum(t_step) / len(t_step)
    per_group_rect = sum(t_rect) / len(t_rect)
    us = (per_group_step + per_group_rect / f) * groups * 1e6
    return {"value": round(us, 1), "unit": "us/step", "cores": cores, "kind": "oracle",
            "sample": (f"{sampled} of {groups} (batch, kv-head) groups at full context: one decode "
                       f"step each (append, select, sparse attend) plus one rectification of "
                       f"{f} rows amortised over {f} steps, scaled to all {groups} groups")}


def measure(args, w, dense: bool) -> dict:
    """Runs the decode loop of workload `w` and returns the result fields."""
    import torch

    import paper_2506_04108_amd as R
    from paper_2506_04108_amd._lib import SelectParams, check, lib
    import workloads.device as WD

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    L0, B, H, Hq, D, b = w.seq_len, w.batch, w.num_kv_heads, w.num_q_heads, w.head_dim, w.block_size
    f = w.rectify_every
    nlay = max(1, args.layers)
    total = args.warmup + args.steps
    per_layer = -(-total // nlay)
    cap = L0 + 2 * per_layer + b + args.cap_pad  # the replay pass appends once more
    cap = -(-cap // b) * b
    stream = torch.cuda.current_stream()
    sptr = stream.cuda_stream
    launch_stream = [sptr]  # the capture stream while a graph is recorded
    lb = lib()

    log(f"[bench] {describe(w, nlay, dense)}; capacity {cap}")
    t_gen = time.perf_counter()
    layers = []
    for li in range(nlay):
        K, V, scale, plant = WD.caches(w, cap, li, dev)
        mb = cap // b
        table = None
        if args.paged:
            # Serving layout: the layer's blocks scattered over a shuffled page pool.
            g = torch.Generator(device=dev)
            g.manual_seed(4108 + li)
            table = torch.randperm(B * mb, generator=g, device=dev).to(torch.int32).view(B, mb)
            K, V = (WD.to_pages(X, table, b) for X in (K, V))
        cache = R.KVCache(K, V, torch.empty((B, H, mb, D), dtype=torch.bfloat16, device=dev),
                          torch.empty((B, H, mb, D), dtype=torch.bfloat16, device=dev), b, table)
        lens = torch.full((B,), L0, dtype=torch.int32, device=dev)
        R.block_summarize(cache, lens)
        q, k, v = WD.step_inputs(w, per_layer, li, scale, plant, dev)
        layers.append(dict(cache=cache, desc=cache.desc(), lens=lens, q=q, k=k, v=v, steps=0))
    torch.cuda.synchronize()
    log(f"[bench] inputs ready in {time.perf_counter() - t_gen:.1f}s")

    mcap = cap // b
    if dense:
        n_cap = mcap
    else:
        n_cap = R.num_selected(mcap, w.sparsity, w.min_blocks, w.n_local)
    idx = torch.empty((B, H, n_cap), dtype=torch.int32, device=dev)
    nsel = torch.empty((B, H), dtype=torch.int32, device=dev)
    out = torch.empty((B, Hq, D), dtype=torch.float32, device=dev)
    lse = torch.empty((B, Hq), dtype=torch.float32, device=dev)
    splits = args.splits if args.splits > 0 else R.decode_num_splits(B, H, n_cap, b)
    # One selection workspace per layer: besides scratch it carries the
    # digit-window hint of the layer's previous call.
    ws_sels = [torch.zeros(max(lb.resa_select_workspace_size(B, H, cap, b), 256), dtype=torch.uint8,
                           device=dev) for _ in range(nlay)]
    ws_dec = torch.zeros(lb.resa_decode_workspace_size(B, H, Hq, n_cap, b, splits), dtype=torch.uint8,
                         device=dev)
    # Fused steps: one workspace per layer as well (it holds the selection hint).
    ws_steps = [torch.zeros(max(lb.resa_step_workspace_size(B, H, Hq, cap - 1, b, n_cap, splits), 256),
                            dtype=torch.uint8, device=dev) for _ in range(nlay)] if args.mode == "step" else []
    ws_rec = torch.zeros(lb.resa_rectify_workspace_size(B, H, Hq, f, cap), dtype=torch.uint8, device=dev)
    rout = torch.empty((B, Hq, f, D), dtype=torch.float32, device=dev)
    params = SelectParams(w.sparsity, w.min_blocks, w.n_local)
    sm = 1.0 / math.sqrt(D)

    # Dense baseline: every block id in order, count = M (decode only).
    if dense:
        all_idx = torch.arange(n_cap, dtype=torch.int32, device=dev).repeat(B, H, 1).contiguous()

    # Rectification rows are prepared ahead (inputs, not timed work).
    rect_inputs = {}
    for li, ly in enumerate(layers):
        for s in range(f, per_layer + 1, f):
            lo = s - f
            k_last = ly["k"][lo:s].permute(1, 2, 0, 3).contiguous()
            v_last = ly["v"][lo:s].permute(1, 2, 0, 3).contiguous()
            rect_inputs[li, s] = WD.rectify_rows(w, k_last, v_last, f, 100 * li + s, dev)
    torch.cuda.synchronize()

    # Busy burst before each timed region (--burst-ms, 5 ms by default): the
    # GPU's clocks drop during the host synchronisations that separate the
    # regions, and a short region (say 20 steps, 2 ms) would be timed while
    # they ramp back up (measured: decode 44.2 against 42.0 us). Reads of a
    # 256 MiB buffer (about 40 us each) keep the GPU busy up to the region's
    # first launch, as in a serving loop that runs steps back to back.
    burst_buf = torch.zeros(2 ** 27, dtype=torch.int16, device=dev) if args.burst_ms > 0 else None
    burst_sink = torch.zeros(1, dtype=torch.int32, device=dev)

    def burst():
        if burst_buf is None:
            return
        for _ in range(max(1, int(args.burst_ms * 1000 / 40))):
            check(lb.resa_stream_read(burst_buf.data_ptr(), burst_buf.numel() * 2, burst_sink.data_ptr(),
                                      1, 256, launch_stream[0]))

    # Per-step selections are kept so the per-kernel timing pass below can
    # replay each launch with the arguments it had in the timed loop.
    idx_all = torch.empty((args.steps, B, H, n_cap), dtype=torch.int32, device=dev)
    nsel_all = torch.empty((args.steps, B, H), dtype=torch.int32, device=dev)
    calls = []  # (phase, layer, step-in-layer, timed-step, Lcur)

    def launch(phase, li, s, t, Lcur):
        ly = layers[li]
        d = C.byref(ly["desc"])
        ids, ns = (idx_all[t], nsel_all[t]) if t >= 0 else (idx, nsel)
        if phase == "step":
            check(lb.resa_decode_step(d, ly["k"][s].data_ptr(), ly["v"][s].data_ptr(), ly["q"][s].data_ptr(),
                                      Hq, ly["lens"].data_ptr(), Lcur, C.byref(params), ids.data_ptr(),
                                      ns.data_ptr(), n_cap, splits, sm, out.data_ptr(), lse.data_ptr(),
                                      ws_steps[li].data_ptr(), ws_steps[li].numel(), launch_stream[0]))
        elif phase == "append_select":
            check(lb.resa_append_select(d, ly["k"][s].data_ptr(), ly["v"][s].data_ptr(), ly["q"][s].data_ptr(),
                                        Hq, ly["lens"].data_ptr(), Lcur, C.byref(params), ids.data_ptr(),
                                        ns.data_ptr(), n_cap, None, ws_sels[li].data_ptr(), ws_sels[li].numel(), launch_stream[0]))
        elif phase == "append":
            check(lb.resa_append_kv(d, ly["k"][s].data_ptr(), ly["v"][s].data_ptr(),
                                    ly["lens"].data_ptr(), Lcur, launch_stream[0]))
        elif phase == "select":
            check(lb.resa_select_blocks(d, ly["q"][s].data_ptr(), Hq, ly["lens"].data_ptr(), Lcur + 1,
                                        C.byref(params), ids.data_ptr(), ns.data_ptr(), n_cap, None,
                                        ws_sels[li].data_ptr(), ws_sels[li].numel(), launch_stream[0]))
        elif phase == "decode":
            if dense:
                ids = all_idx
            check(lb.resa_sparse_decode(d, ly["q"][s].data_ptr(), Hq, ly["lens"].data_ptr(),
                                        ids.data_ptr(), ns.data_ptr(), n_cap, splits, sm, out.data_ptr(),
                                        lse.data_ptr(), ws_dec.data_ptr(), ws_dec.numel(), launch_stream[0]))
        else:
            qf, kf, vf = rect_inputs[li, s + 1]
            check(lb.resa_dense_rectify(d, qf.data_ptr(), kf.data_ptr(), vf.data_ptr(), Hq, f,
                                        ly["lens"].data_ptr(), None, Lcur + 1, sm, rout.data_ptr(), None, 1,
                                        ws_rec.data_ptr(), ws_rec.numel(), launch_stream[0]))

    def step(t):
        """One decode step (t >= 0: timed step t, its selection kept)."""
        li = step.count % nlay
        step.count += 1
        ly = layers[li]
        s = ly["steps"]
        Lcur = L0 + s
        if dense:
            seq = ["append", "decode"]
        elif args.mode == "three":
            seq = ["append", "select", "decode"]
        elif args.mode == "step":
            seq = ["step"]
        else:
            seq = ["append_select", "decode"]
        if not dense and (s + 1) % f == 0:
            seq.append("rectify")
        if dense:
            (nsel_all[t] if t >= 0 else nsel).fill_(-(-(Lcur + 1) // b))
        for ph in seq:
            launch(ph, li, s, t, Lcur)
            if t >= 0:
                calls.append((ph, li, s, t, Lcur))
        ly["steps"] = s + 1
        return Lcur + 1

    step.count = 0
    for _ in range(args.warmup):
        step(-1)
    if args.copy_probe:
        # One plain device copy of known size: the reference that scales the
        # FETCH_SIZE / WRITE_SIZE counters in a rocprofv3 --pmc run.
        src = torch.empty(args.copy_probe // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        del src, dst
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    lens_seen = []
    if args.graph:
        # The timed steps are recorded once into a HIP graph (recording runs
        # nothing), replayed once to warm up, and after the lengths are put
        # back, replayed again under the events: the same launches with the
        # same host bounds, without per-launch host work. The second replay
        # rewrites the same rows; summaries already hold them, so the
        # selections can differ slightly from an eager run, not the amount
        # of work.
        lens0 = [ly["lens"].clone() for ly in layers]
        graph = torch.cuda.CUDAGraph()
        cap_stream = torch.cuda.Stream()
        cap_stream.wait_stream(stream)
        torch.cuda.synchronize()
        with torch.cuda.graph(graph, stream=cap_stream):
            launch_stream[0] = cap_stream.cuda_stream
            for t in range(args.steps):
                lens_seen.append(step(t))
        launch_stream[0] = sptr
        graph.replay()
        torch.cuda.synchronize()
        for ly, l0 in zip(layers, lens0):
            ly["lens"].copy_(l0)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        burst()
        e0.record(stream)
        graph.replay()
        e1.record(stream)
    else:
        t0 = time.perf_counter()
        burst()
        e0.record(stream)
        for t in range(args.steps):
            lens_seen.append(step(t))
        e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gpu_ms = e0.elapsed_time(e1)

    # Per-kernel timing: every launch of one phase from the timed loop is
    # replayed back to back, bracketed by two events on the launch stream, so
    # the average is the kernel's own duration (no host launch gaps and no
    # event packets between launches). Select, decode and rectify only read
    # the cache (rectify rewrites the rows it was given); the fused
    # append + select replay, last, appends the same tokens once more into the
    # capacity kept for it (so does the fused step's replay). The plain append
    # kernel (--mode three, --dense) runs for less time than one host launch
    # takes, so a replay would time the host; its duration is taken from a
    # kernel trace instead. With fused steps, the standalone decode kernel is
    # also timed on the selections the steps made ("decode_alone", not part
    # of the step).
    phase_us = {}
    for ph in ("select", "decode", "decode_alone", "rectify", "append_select", "step"):
        cs = [c for c in calls if c[0] == ("step" if ph == "decode_alone" else ph)]
        if not cs:
            continue
        a, z = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        burst()
        a.record(stream)
        for _, li, s, t, _ in cs:
            # The host length bound must hold for the cache as it is now.
            n = layers[li]["steps"]
            if ph in ("append_select", "step"):
                launch(ph, li, s, t, L0 + n)
                layers[li]["steps"] = n + 1
            else:
                launch("decode" if ph == "decode_alone" else ph, li, s, t, L0 + n - 1)
        z.record(stream)
        torch.cuda.synchronize()
        phase_us[ph] = a.elapsed_time(z) * 1e3 / len(cs)

    # Rectification (Alg. 1: every f-th step of a layer) enters the step at
    # its amortised rate, one call per f steps (the 1/f term of Eq. 6), for
    # any number of timed steps: the calls made inside the timed window are
    # taken out of the timed GPU time at their measured per-call duration and
    # the per-call duration / f is added back. When the window holds no call
    # (fewer than f steps per layer), one call per layer is timed on its own,
    # on the cache as the loop left it, with rows of the layer's decode inputs.
    n_rect_in = sum(1 for c in calls if c[0] == "rectify")
    rect_how = None
    if not dense:
        if "rectify" in phase_us:
            rect_how = "inside the timed window"
        else:
            reps = 1
            rin = []
            for li, ly in enumerate(layers):
                pick = torch.arange(f, device=dev) % per_layer
                k_last = ly["k"][pick].permute(1, 2, 0, 3).contiguous()
                v_last = ly["v"][pick].permute(1, 2, 0, 3).contiguous()
                rin.append(WD.rectify_rows(w, k_last, v_last, f, 7919 + li, dev))
            torch.cuda.synchronize()

            def rect_call(li):
                ly = layers[li]
                qf, kf, vf = rin[li]
                Lc = L0 + ly["steps"]
                check(lb.resa_dense_rectify(C.byref(ly["desc"]), qf.data_ptr(), kf.data_ptr(),
                                            vf.data_ptr(), Hq, f, ly["lens"].data_ptr(), None, Lc, sm,
                                            rout.data_ptr(), None, 1, ws_rec.data_ptr(),
                                            ws_rec.numel(), sptr))
            a, z = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            burst()
            a.record(stream)
            for _ in range(reps):
                for li in range(nlay):
                    rect_call(li)
            z.record(stream)
            torch.cuda.synchronize()
            phase_us["rectify"] = a.elapsed_time(z) * 1e3 / (reps * nlay)
            rect_how = (f"timed separately ({reps} call per layer, as the in-window replay): fewer "
                        "than f steps per layer in the window")
    t_rect = phase_us.get("rectify", 0.0)
    timed_us = gpu_ms * 1e3 / args.steps
    step_us = (gpu_ms * 1e3 - n_rect_in * t_rect) / args.steps + (t_rect / f if not dense else 0.0)

    # Algorithmic bytes of each launch: the selected blocks' K and V rows
    # (decode), plus the kmin / kmax summaries of every block (fused step).
    bytes_dec, bytes_sum = [], []
    for L in lens_seen:
        M = -(-L // b)
        n = M if dense else R.num_selected(M, w.sparsity, w.min_blocks, w.n_local)
        bytes_dec.append(B * H * n * b * D * 2 * 2)
        bytes_sum.append(B * H * M * D * 2 * 2)
    avg_bytes = sum(bytes_dec) / len(bytes_dec)
    avg_sum = sum(bytes_sum) / len(bytes_sum)
    import workloads as W
    plain = w == W.WORKLOADS.get(w.name) and not (dense or args.paged or args.mode == "three")

    def roof(kernel, profile, nbytes, us):
        gbs = nbytes / (us * 1e-6) / 1e9
        return {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(gbs / HBM_PEAK_GBS, 4),
                "traffic": traffic_from_profile(kernel, f"{profile}_{w.name.replace('_', '')}"
                                                if plain else None),
                "kernel": kernel, "avg_launch_us": round(us, 3), "bytes_per_launch": int(nbytes)}

    dec_key = "decode_alone" if "decode_alone" in phase_us else "decode"
    dec_roof = roof("k_decode", "sparse_decode", avg_bytes, phase_us[dec_key])
    if "step" in phase_us:
        roofline = roof("k_step", "decode_step", avg_bytes + avg_sum, phase_us["step"])
    else:
        roofline = dec_roof
    ms_per_step = step_us / 1e3
    n_calls = {ph: sum(1 for c in calls if c[0] == ph) for ph in phase_us}
    per_step = {k: round(v * n_calls[k] / args.steps, 2) for k, v in phase_us.items() if k != "rectify"}
    rect = None
    if not dense:
        per_step["rectify"] = round(t_rect / f, 2)
        # Rectification roofline: every group's K and V read once (L x 512 B per
        # group at the mean length of the calls) and the matrix work of causal
        # attention, 4 * 128 flops per (query head, window row, visible key).
        Lr = (sum(c[4] + 1 for c in calls if c[0] == "rectify") / n_rect_in) if n_rect_in else \
            (L0 + sum(ly["steps"] for ly in layers) / nlay)
        r_bytes = B * H * Lr * D * 2 * 2
        visible = f * (Lr - f) + f * (f + 1) / 2
        r_flops = 4.0 * D * Hq * B * visible
        r_gbs = r_bytes / (t_rect * 1e-6) / 1e9
        r_tf = r_flops / (t_rect * 1e-6) / 1e12
        rect = {"us_per_call": round(t_rect, 2), "every": f, "us_per_step": round(t_rect / f, 2),
                "calls_in_window": n_rect_in, "timing": rect_how,
                "hbm": {"achieved": round(r_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                        "frac": round(r_gbs / HBM_PEAK_GBS, 4), "bytes_per_call": int(r_bytes)},
                "mfma": {"achieved": round(r_tf, 1), "peak": MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                         "frac": round(r_tf / MFMA_PEAK_TFLOPS, 4), "flops_per_call": r_flops}}
    res = {
        "metric": METRIC,
        "value": round(step_us, 2),
        "unit": "us/step",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": describe(w, nlay, dense), "mode": args.mode, "batch": B, "q_heads": Hq,
                   "kv_heads": H,
                   "head_dim": D, "context_start": L0, "block_size": b,
                   "sparsity": None if dense else w.sparsity, "min_tokens": w.min_tokens,
                   "rectify_every": f, "decode_splits": splits, "layers_rotated": nlay,
                   "hip_graph": bool(args.graph), "paged": bool(args.paged)},
        "roofline": roofline,
        "decode_roofline": dec_roof,
        "kernel_us_per_launch": {k: round(v, 2) for k, v in phase_us.items()},
        "kernel_us_per_step": per_step,
        "rectify_roofline": rect,
        "timed_gpu_us_per_step": round(timed_us, 2),
        "wall_us_per_step": round(wall * 1e6 / args.steps, 2),
    }
    if args.stream_probe > 0:
        res["stream_read_ceiling"] = stream_ceiling(lb, check, dev, stream, args.stream_probe)
        res["decode_roofline"]["frac_of_stream_ceiling"] = round(
            dec_roof["achieved"] / res["stream_read_ceiling"]["achieved"], 4)
    return res


def stream_ceiling(lb, check, dev, stream, nbytes) -> dict:
    """HBM read ceiling on this GPU: resa_stream_read over a buffer of
    `nbytes` (larger than the last-level cache) at a few grid sizes, the
    median of 5 timed reads each; the best grid is reported."""
    import torch
    buf = torch.zeros(nbytes // 2, dtype=torch.bfloat16, device=dev)
    sink = torch.zeros(1, dtype=torch.int32, device=dev)
    best = None
    for wgs in (256, 512, 1024, 2048):
        def run():
            check(lb.resa_stream_read(buf.data_ptr(), buf.numel() * 2, sink.data_ptr(), 1, wgs,
                                      stream.cuda_stream))
        for _ in range(2):
            run()
        times = []
        for _ in range(5):
            a, z = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            run()
            z.record(stream)
            torch.cuda.synchronize()
            times.append(a.elapsed_time(z) * 1e3)
        us = sorted(times)[2]
        if best is None or us < best[0]:
            best = (us, wgs)
    us, wgs = best
    gbs = buf.numel() * 2 / (us * 1e-6) / 1e9
    del buf
    return {"achieved": round(gbs, 1), "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4),
            "bytes": int(nbytes), "us": round(us, 2), "workgroups": wgs, "kernel": "k_stream_read"}


def breakdown(args) -> dict:
    """Per-kernel latency of one decode step at 16K, 64K and 256K context
    (batch 8, the 64K workload's recipe), against a dense decode over every
    block: sparse estimation (append + select), attention (decode) and
    rectification (one call amortised over f steps)."""
    import workloads as W
    rows = []
    args.mode = "two"  # estimation and attention as separate kernels
    for L in (16384, 65536, 262144):
        w = W.LONG_64K.with_(seq_len=L)
        sp = measure(args, w, False)
        dn = measure(args, w, True)
        k = sp["kernel_us_per_launch"]
        f = w.rectify_every
        est, att, rect = k["append_select"], k["decode"], k["rectify"] / f
        tot = est + att + rect
        rows.append({"context": L, "estimation_us": round(est, 2), "attention_us": round(att, 2),
                     "rectification_us": round(rect, 2),
                     "rectification_share": round(rect / tot, 4),
                     "resa_kernel_us": round(tot, 2), "dense_decode_us": dn["kernel_us_per_launch"]["decode"],
                     "speedup_vs_dense": round(dn["kernel_us_per_launch"]["decode"] / tot, 3),
                     "decode_hbm_frac": sp["roofline"]["frac"],
                     "dense_hbm_frac": dn["roofline"]["frac"]})
    return {"breakdown": rows, "workload": describe(W.LONG_64K, args.layers, False)}


def sweep(args) -> dict:
    """The 64K batch-8 sweep (block size 16/32/64 x sparsity 0.8/0.9/0.95 x
    rectify interval 16/32/64, N(0, 1) caches with 1 % planted blocks) and,
    per block size, dense decoding over every block. Each point runs 2 f
    timed steps over two layer caches (so each layer is rectified once);
    us_per_step is the GPU time of those steps, rectification included."""
    import workloads as W
    rows = []
    args.mode, args.layers = "two", 2
    for w in W.sweep_points():
        f = w.rectify_every
        args.steps, args.warmup = 2 * f, 4
        r = measure(args, w, False)
        k = r["kernel_us_per_launch"]
        rows.append({"block_size": w.block_size, "sparsity": w.sparsity, "f": f,
                     "us_per_step": r["value"],
                     "estimation_us": round(k["append_select"], 2), "attention_us": round(k["decode"], 2),
                     "rectification_us_per_step": round(k.get("rectify", 0.0) / f, 2),
                     "decode_hbm_frac": r["roofline"]["frac"]})
        log(f"[bench] sweep b={w.block_size} s={w.sparsity} f={f}: {r['value']} us/step")
    dense = {}
    for b in (16, 32, 64):
        w = W.SWEEP_64K.with_(block_size=b, planted_per_head=0)
        args.steps, args.warmup = 32, 4
        r = measure(args, w, True)
        dense[b] = {"us_per_step": r["value"], "decode_us": r["kernel_us_per_launch"]["decode"],
                    "decode_hbm_frac": r["roofline"]["frac"]}
    for row in rows:
        row["speedup_vs_dense"] = round(dense[row["block_size"]]["us_per_step"] / row["us_per_step"], 3)
    return {"sweep": rows, "dense": dense, "workload": describe(W.SWEEP_64K, 2, False)}



def prefill(args) -> dict:
    """Prefill through the rectification call (Alg. 1, prefill step): a prompt
    chunk of f rows is written into the cache, its queries attend causally to
    the cache before it and to themselves, and its block summaries are built.
    Cases: the last 4096-token chunk of a 64K prompt at batch 8, and whole
    8K and 32K prompts (f = L). The rate counts the matrix work of causal
    attention, 4 * 128 flops per (query head, row, visible key)."""
    import torch

    import paper_2506_04108_amd as R
    import workloads as W
    import workloads.device as WD

    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    rows = []
    for name, B, L, f in (("chunk4096_ctx65536_batch8", 8, 65536, 4096),
                          ("prompt8192_batch8", 8, 8192, 8192),
                          ("prompt32768_batch1", 1, 32768, 32768)):
        w = W.LONG_64K.with_(batch=B, seq_len=L)
        H, Hq, D, b = w.num_kv_heads, w.num_q_heads, w.head_dim, w.block_size
        K, V, scale, plant = WD.caches(w, L, 0, dev)
        mb = L // b
        cache = R.KVCache(K, V, torch.empty((B, H, mb, D), dtype=torch.bfloat16, device=dev),
                          torch.empty((B, H, mb, D), dtype=torch.bfloat16, device=dev), b)
        lens = torch.full((B,), L, dtype=torch.int32, device=dev)
        if f < L:
            R.block_summarize(cache, lens)
        qf, kf, vf = WD.rectify_rows(w, K[:, :, L - f:], V[:, :, L - f:], f, 7, dev)
        out = torch.empty((B, Hq, f, D), dtype=torch.float32, device=dev)
        lse = torch.empty((B, Hq, f), dtype=torch.float32, device=dev)
        ws = R.Workspace(dev)
        call = lambda: R.dense_rectify(cache, qf, kf, vf, lens, L, out=out, lse=lse, workspace=ws)
        for _ in range(3):
            call()
        torch.cuda.synchronize()
        reps = 10 if f * L * B < 2 ** 31 else 4
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            call()
        e1.record(stream)
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / reps
        visible = f * (L - f) + f * (f + 1) // 2
        flops = 4.0 * D * Hq * B * visible
        tf = flops / (us * 1e-6) / 1e12
        log(f"[bench] prefill {name}: {us:.1f} us, {tf:.1f} TFLOP/s")
        rows.append({"case": name, "batch": B, "context": L, "f": f, "us_per_call": round(us, 2),
                     "tflops": round(tf, 1), "peak": MFMA_PEAK_TFLOPS,
                     "frac": round(tf / MFMA_PEAK_TFLOPS, 4)})
        del K, V, cache, qf, kf, vf, out, lse, ws
        torch.cuda.empty_cache()
    return {"prefill": rows, "unit": "TFLOP/s", "bound": "mfma", "dtype": "bf16/f16 in, f32 acc"}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the library has no "
              "multi-GPU path.", file=sys.stderr)
        sys.exit(2)
    import torch
    torch.cuda.set_device(0)
    if args.breakdown:
        print(json.dumps(breakdown(args)), flush=True)
        return
    if args.sweep:
        print(json.dumps(sweep(args)), flush=True)
        return
    if args.prefill:
        print(json.dumps(prefill(args)), flush=True)
        return
    w = workload_of(args)
    res = measure(args, w, args.dense)
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a bounded sample")
        res["cpu_baseline"] = cpu_baseline(w, args.cpu_budget)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
