"""Benchmark of the KV-composition hot path on one MI355X.

One step = one full composition of a 65,536-token, 36-layer Qwen2.5-VL-3B
shaped bf16 cache (32 chunks x 2048 tokens, 16 query / 2 KV heads, head dim
128, mRoPE sections 16/24/24) at rho = 0.1:
  compose_rebase_k -> score_deviation_topk -> 36 x selective_attend_scatter
(one call per layer, the model's layer-by-layer order).  The caches are
restored from a pristine copy before every step, outside the timed region
(re-basing and scattering are in place); each step is bracketed by a device
synchronisation and HIP events on the stream the library launches on.

Inputs are synthetic and seeded (torch's device generator): stored keys and
values ~ N(0,1) (a rotation of an isotropic Gaussian is again N(0,1), so the
stored post-rotary keys are drawn directly), fresh queries ~ N(0,1), fresh
keys = re-based stored keys + s_t z and fresh values = stored values + s_t z'
with z, z' ~ N(0, 0.1^2) and s_t ~ LogNormal(0,1) per token.  The re-based
keys used to build the fresh keys come from one untimed call of the library's
own compose_rebase_k during set-up.

Prints ONE JSON line on stdout; progress goes to stderr.
"""
import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=10)
    p.add_argument("--warmup", type=int, default=2)
    p.add_argument("--workload", default="long65k")
    p.add_argument("--rho", type=float, default=None)
    p.add_argument("--rho1-steps", type=int, default=2, help="steps timed at rho = 1.0 (0: skip)")
    p.add_argument("--cpu-baseline", type=int, default=1, help="time the CPU oracle on a sample (0: skip)")
    p.add_argument("--batched-layers", type=int, default=0,
                   help="one selective_attend_scatter call over all layers instead of one per layer")
    p.add_argument("--fused-rope-steps", type=int, default=6,
                   help="steps of each, alternating: selective_attend_scatter_rope (pre-rotary fresh rows, "
                        "rotated at the global coordinates) and the plain call (0: skip)")
    p.add_argument("--gemm-context", type=int, default=1,
                   help="also time the vendor library's bf16 GEMM on this GPU, as context for the MFMA figure (0: skip)")
    p.add_argument("--load-steps", type=int, default=3,
                   help="steps of the chunks' load from page-locked host memory with the re-basing as each "
                        "chunk lands, against plain copies and copies followed by the re-basing (0: skip)")
    p.add_argument("--paged-steps", type=int, default=3,
                   help="steps also timed on the cache held as one buffer per chunk (0: skip)")
    p.add_argument("--batched-steps", type=int, default=3,
                   help="steps also timed with one batched attention call over all layers (0: skip)")
    p.add_argument("--graph-steps", type=int, default=3,
                   help="steps of the per-layer composition captured once into a HIP graph and replayed (0: skip)")
    p.add_argument("--oracle-full", choices=("none", "tiny", "qwen8k"), default="none",
                   help="time the CPU oracle's whole composition of a small workload (all layers, "
                        "no extrapolation) and print one JSON line; needs no GPU")
    p.add_argument("--sweep", choices=("none", "rebase", "attention"), default="none",
                   help="rebase: 8k/65k/262k-token K caches with and without a cache flush, and the "
                        "per-token (scalar re-basing) kernel on the 65k cache; "
                        "attention: the 32k-token cache at rho in {0.05, 0.1, 0.2, 0.5, 1}")
    return p.parse_args()


class Inputs:
    def __init__(self, w, torch, binding, synth):
        dev = "cuda"
        bf = torch.bfloat16
        L, Hkv, Hq, T, D, n = w.n_layers, w.n_kv_heads, w.n_q_heads, w.n_tokens, w.head_dim, w.n_candidates
        cs1 = w.cs1
        self.geo = binding.Geo.from_workload(w)
        self.offsets = synth.chunk_offsets(w)
        log(f"[bench] generating inputs: L={L} T={T} n={n}")
        self.K0 = torch.empty((L, Hkv, T, D), dtype=bf, device=dev)
        self.V0 = torch.empty((L, Hkv, T, D), dtype=bf, device=dev)
        self.QF = torch.empty((L, Hq, n, D), dtype=bf, device=dev)
        self.KF = torch.empty((L, Hkv, n, D), dtype=bf, device=dev)
        self.VF = torch.empty((L, Hkv, n, D), dtype=bf, device=dev)
        s = synth.torch_token_scale(w, dev)[None, :, None]
        for layer in range(L):
            self.K0[layer] = synth.torch_normal((Hkv, T, D), w.seed, 0, synth.TAG_K, layer, dev, bf)
            self.V0[layer] = synth.torch_normal((Hkv, T, D), w.seed, 0, synth.TAG_V, layer, dev, bf)
            self.QF[layer] = synth.torch_normal((Hq, n, D), w.seed, 2, synth.TAG_Q, layer, dev, bf)
        kreb = self.K0.clone()
        binding.compose_rebase_k(self.geo, kreb, self.offsets)
        for layer in range(L):
            zk = synth.torch_normal((Hkv, n, D), w.seed, 1, synth.TAG_ZK, layer, dev, torch.float32, 0.1)
            zv = synth.torch_normal((Hkv, n, D), w.seed, 1, synth.TAG_ZV, layer, dev, torch.float32, 0.1)
            self.KF[layer] = (kreb[layer, :, cs1:].float() + s * zk).to(bf)
            self.VF[layer] = (self.V0[layer, :, cs1:].float() + s * zv).to(bf)
        del kreb
        loc = synth.local_coords(w).astype(np.int64)
        glob = loc.copy()
        cs = w.chunk_start
        for c in range(w.n_chunks):
            glob[cs[c]:cs[c + 1]] += self.offsets[c]
        self.coords = torch.from_numpy(glob.astype(np.int32)).to(dev)   # global coordinates [T, 3]
        self.K = self.K0.clone()
        self.V = self.V0.clone()
        torch.cuda.synchronize()


def busy_gpu(torch):
    """A ~0.2 ms spin kernel ahead of a timed region (outside it): the GPU is still busy while the
    host enqueues the first launches of the region, so the region's events and the per-kernel
    trace events measure device work, not the host's enqueue latency."""
    torch.cuda._sleep(400_000)


def run_compose(inp, w, rho, binding, torch, out, lse, sel, scores, ws, batched, fused=False, paged=False):
    b = binding
    if paged:   # the same composition on the cache held as one buffer per chunk
        b.compose_rebase_k_paged(inp.geo, inp.Kc, inp.offsets)
        k = b.score_deviation_topk_paged(inp.geo, inp.Kc, w.score_layer, inp.KF[w.score_layer], rho, scores, sel)
        for layer in range(w.n_layers):
            b.selective_attend_scatter_paged(inp.geo, inp.Kc, inp.Vc, layer, layer + 1, sel, k, inp.QF, inp.KF,
                                             inp.VF, out, lse, ws)
        return k
    b.compose_rebase_k(inp.geo, inp.K, inp.offsets)
    k = b.score_deviation_topk(inp.geo, inp.K, w.score_layer, inp.KF[w.score_layer], rho, scores, sel)
    if fused:   # QF and KF taken as the pre-rotary fresh rows (N(0, 1) either way)
        for layer in range(w.n_layers):
            b.selective_attend_scatter_rope(inp.geo, inp.K, inp.V, layer, layer + 1, sel, k, inp.QF, inp.KF,
                                            inp.VF, inp.coords, out, lse, ws)
    elif batched:
        b.selective_attend_scatter(inp.geo, inp.K, inp.V, 0, w.n_layers, sel, k, inp.QF, inp.KF, inp.VF,
                                   out, lse, ws)
    else:
        for layer in range(w.n_layers):
            b.selective_attend_scatter(inp.geo, inp.K, inp.V, layer, layer + 1, sel, k, inp.QF, inp.KF,
                                       inp.VF, out, lse, ws)
    return k


def host_info():
    threads = None
    try:
        from threadpoolctl import threadpool_info
        threads = max((i.get("num_threads", 1) for i in threadpool_info()), default=1)
    except Exception:
        threads = os.cpu_count()
    cpu_model = None
    try:
        with open("/proc/cpuinfo") as f:
            cpu_model = next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")), None)
    except OSError:
        pass
    return threads, cpu_model


def oracle_full(name):
    """The CPU oracle's whole composition of a small workload (every layer, no
    extrapolation): re-basing, scoring, selection, and the scatter and attention
    of every layer, timed after the inputs are built."""
    import oracle
    from paper_2607_19547_amd import synth
    w = synth.WORKLOADS[name]
    d = oracle.inputs.build(w)
    args = (w.dtype, w.head_dim, w.sections, w.base, d["chunk_start"], d["chunk_offsets"], d["k_stored"],
            d["v_stored"], d["q_fresh"], d["k_fresh"], d["v_fresh"], w.rho, w.score_layer)
    reps = 20 if name == "tiny" else 1
    times = []
    for _ in range(reps):
        t0 = time.perf_counter()
        oracle.compose.compose(*args)
        times.append(time.perf_counter() - t0)
    threads, cpu_model = host_info()
    print(json.dumps({"oracle_full": {"workload": name, "rho": w.rho, "n_layers": w.n_layers, "n_tokens": w.n_tokens,
                                      "median_s": float(np.median(times)), "reps": reps, "cores": threads,
                                      "host_cpus": os.cpu_count(), "cpu_model": cpu_model,
                                      "kind": "oracle", "dtype": "f64"}}), flush=True)


def main():
    args = parse()
    if args.oracle_full != "none":
        return oracle_full(args.oracle_full)
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the library has no "
              f"multi-GPU path: run with --gpus 1", file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_2607_19547_amd import binding, synth
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    binding.lib()
    if args.sweep == "rebase":
        return sweep_rebase(args, binding, synth, torch)
    if args.sweep == "attention":
        return sweep_attention(args, binding, synth, torch)
    w = synth.WORKLOADS[args.workload]
    rho = w.rho if args.rho is None else args.rho
    inp = Inputs(w, torch, binding, synth)
    result = bench_rho(inp, w, rho, args.steps, args.warmup, binding, torch, bool(args.batched_layers),
                       untraced_steps=args.steps)
    rho1 = None
    if args.rho1_steps > 0 and rho != 1.0:
        rho1 = bench_rho(inp, w, 1.0, args.rho1_steps, 1, binding, torch, bool(args.batched_layers))
    other = None
    if args.batched_steps > 0:  # the other launch mode, for comparison
        other = bench_rho(inp, w, rho, args.batched_steps, 1, binding, torch, not args.batched_layers)
    fused = None
    if args.fused_rope_steps > 0:
        fused = bench_fused_vs_plain(inp, w, rho, args.fused_rope_steps, binding, torch)
    paged = None
    if args.paged_steps > 0:
        paged = bench_rho(inp, w, rho, args.paged_steps, 1, binding, torch, False, paged=True)
    graph = bench_graph(inp, w, rho, args.graph_steps, binding, torch) if args.graph_steps > 0 else None
    load = bench_load(inp, w, args.load_steps, binding, torch) if args.load_steps > 0 else None
    gemm = gemm_context(torch) if args.gemm_context else None
    cpu = cpu_baseline(w, rho) if args.cpu_baseline else None
    emit(args, w, rho, result, rho1, cpu, other, fused, paged, gemm, graph, load)


def bench_load(inp, w, steps, binding, torch):
    """The cache's chunks (K and V, [L, H_kv, len_c, D] each) from page-locked host memory into device
    chunk buffers: plain copies; compose_load_rebase_k_paged (copies on a second stream, the keys
    first, re-based on the compute stream while the values are in transfer); and copies followed by
    compose_rebase_k_paged.  Medians of HIP events on the compute stream (PCIe included)."""
    b = binding
    cs = w.chunk_start
    n_chunks = len(cs) - 1
    kh = [inp.K0[:, :, cs[c]:cs[c + 1]].contiguous().cpu().pin_memory() for c in range(n_chunks)]
    vh = [inp.V0[:, :, cs[c]:cs[c + 1]].contiguous().cpu().pin_memory() for c in range(n_chunks)]
    kd = [torch.empty_like(x, device="cuda") for x in kh]
    vd = [torch.empty_like(x, device="cuda") for x in vh]
    nbytes = sum(x.numel() * x.element_size() for x in kh + vh)
    stream = torch.cuda.current_stream()
    copy = torch.cuda.Stream()
    off = inp.offsets

    def plain():
        for d, h in zip(kd + vd, kh + vh):
            d.copy_(h, non_blocking=True)

    def fused():
        b.compose_load_rebase_k_paged(inp.geo, kd, vd, kh, vh, off, copy_stream=copy.cuda_stream)

    def serial():
        plain()
        b.compose_rebase_k_paged(inp.geo, kd, off)

    res = {}
    for name, fn in (("copy", plain), ("load_rebase", fused), ("copy_then_rebase", serial)):
        fn()  # (warm)
        torch.cuda.synchronize()
        res[name], _ = _events(torch, stream, fn, steps)
    fused()
    torch.cuda.synchronize()
    ref = [x.cuda() for x in kh]
    b.compose_rebase_k_paged(inp.geo, ref, off)
    identical = all(torch.equal(x, y) for x, y in zip(kd, ref))
    log(f"[bench] chunk load from host ({nbytes / 1e9:.2f} GB): copies {res['copy']:.3f} ms "
        f"({nbytes / res['copy'] / 1e6:.1f} GB/s), with the re-basing during the load {res['load_rebase']:.3f} ms, "
        f"copies then re-basing {res['copy_then_rebase']:.3f} ms; keys identical to the latter: {identical}")
    del kh, vh, kd, vd, ref
    return dict(res, bytes=nbytes, identical=identical)


def gemm_context(torch, m=8192, n=8192, k=16384, reps=10):
    """bf16 GEMM rate of the vendor BLAS (torch.matmul -> hipBLASLt) on the same GPU and run: the dense
    MFMA rate a tuned library reaches under the same clock and power limits (context only; the
    roofline peak stays the published one)."""
    a = torch.randn(m, k, device="cuda", dtype=torch.bfloat16)
    b = torch.randn(k, n, device="cuda", dtype=torch.bfloat16)
    for _ in range(3):
        c = a @ b
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        c = a @ b
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    tf = 2.0 * m * n * k / (ms / 1e3) / 1e12
    log(f"[bench] vendor bf16 GEMM {m}x{n}x{k}: {ms:.3f} ms, {tf:.1f} TFLOP/s")
    del a, b, c
    return dict(shape=[m, n, k], ms=round(ms, 4), TFLOPs=round(tf, 1))


def bench_fused_vs_plain(inp, w, rho, steps, binding, torch):
    """The fused-RoPE composition and the plain one in alternating steps (plain, fused, plain, ...), so
    that the clock's drift over a run (it follows power and temperature) weighs on both alike; medians
    of each."""
    b = binding
    n = w.n_candidates
    scores = torch.empty(n, dtype=torch.float32, device="cuda")
    sel = torch.empty(n, dtype=torch.int32, device="cuda")
    k = b.score_deviation_topk(inp.geo, inp.K, w.score_layer, inp.KF[w.score_layer], rho, scores, sel)
    out = torch.empty((w.n_layers, w.n_q_heads, k, w.head_dim), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((w.n_layers, w.n_q_heads, k), dtype=torch.float32, device="cuda")
    ws_f = torch.empty(max(b.selective_attend_scatter_rope_workspace(inp.geo, k, 1), 1), dtype=torch.uint8,
                       device="cuda")
    ws_p = torch.empty(max(b.selective_attend_scatter_workspace(inp.geo, k, 1), 1), dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()
    log(f"[bench] rho={rho}: n_sel={k}, fused RoPE and plain in alternating steps, steps {steps} each")
    times = {False: [], True: []}
    trace = {}  # the fused steps' kernels (both kinds are traced alike: the trace's events cost time)
    b.cs_trace_only(("sel_attn_mfma", "plan_scatter", "plan_rope_scatter"))
    for i in range(2 * (steps + 1)):
        fused = i % 2 == 1
        inp.K.copy_(inp.K0)
        inp.V.copy_(inp.V0)
        torch.cuda.synchronize()
        b.cs_trace_reset()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        busy_gpu(torch)
        b.cs_trace_enable(True)
        e0.record(stream)
        run_compose(inp, w, rho, b, torch, out, lse, sel, scores, ws_f if fused else ws_p, False, fused, False)
        e1.record(stream)
        b.cs_trace_enable(False)
        torch.cuda.synchronize()
        step_trace = b.cs_trace_collect()
        if i >= 2:  # the first pair warms up
            times[fused].append(e0.elapsed_time(e1))
            if fused:
                for name, (n_l, ms) in step_trace.items():
                    n0, ms0 = trace.get(name, (0, 0.0))
                    trace[name] = (n0 + n_l, ms0 + ms)
    b.cs_trace_only(None)
    fm, pm = float(np.median(times[True])), float(np.median(times[False]))
    log(f"[bench] rho={rho}: fused RoPE compose median {fm:.3f} ms, plain {pm:.3f} ms (alternating steps)")
    return {"ms": fm, "plain_ms": pm, "trace": trace}


# Kernels whose launches the timed steps trace (the two rooflines); every traced launch costs the GPU a few
# microseconds, so the other kernels' durations come from separate fully traced steps.
ROOFLINE_KERNELS = ("sel_attn_mfma", "rebase_bf16_d128")


def bench_rho(inp, w, rho, steps, warmup, binding, torch, batched, fused=False, paged=False, untraced_steps=0,
              breakdown_steps=2):
    b = binding
    n = w.n_candidates
    scores = torch.empty(n, dtype=torch.float32, device="cuda")
    sel = torch.empty(n, dtype=torch.int32, device="cuda")
    # n_sel is a host-side function of rho and n; one call sizes the buffers
    k = b.score_deviation_topk(inp.geo, inp.K, w.score_layer, inp.KF[w.score_layer], rho, scores, sel)
    out = torch.empty((w.n_layers, w.n_q_heads, k, w.head_dim), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((w.n_layers, w.n_q_heads, k), dtype=torch.float32, device="cuda")
    ws_bytes = (b.selective_attend_scatter_rope_workspace(inp.geo, k, 1) if fused else
                b.selective_attend_scatter_workspace(inp.geo, k, w.n_layers if batched else 1))
    ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()
    log(f"[bench] rho={rho}: n_sel={k}, workspace {ws_bytes / 2**20:.1f} MiB, warmup {warmup}, steps {steps}")

    if paged and not hasattr(inp, "Kc"):
        # one buffer per chunk ([L, H_kv, len_c, D] each), plus pristine copies to restore from
        cs = w.chunk_start
        inp.Kc = [inp.K0[:, :, cs[c]:cs[c + 1]].clone() for c in range(w.n_chunks)]
        inp.Vc = [inp.V0[:, :, cs[c]:cs[c + 1]].clone() for c in range(w.n_chunks)]
        inp.K0c = [x.clone() for x in inp.Kc]
        inp.V0c = [x.clone() for x in inp.Vc]

    def restore():
        if paged:
            for x, x0 in zip(inp.Kc + inp.Vc, inp.K0c + inp.V0c):
                x.copy_(x0)
        else:
            inp.K.copy_(inp.K0)
            inp.V.copy_(inp.V0)

    for _ in range(warmup):
        restore()
        run_compose(inp, w, rho, b, torch, out, lse, sel, scores, ws, batched, fused, paged)
    torch.cuda.synchronize()
    b.cs_trace_reset()
    b.cs_trace_only(ROOFLINE_KERNELS)
    times = []
    wall0 = time.perf_counter()
    for _ in range(steps):
        restore()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        busy_gpu(torch)
        b.cs_trace_enable(True)
        e0.record(stream)
        run_compose(inp, w, rho, b, torch, out, lse, sel, scores, ws, batched, fused, paged)
        e1.record(stream)
        b.cs_trace_enable(False)
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1))
    wall = time.perf_counter() - wall0
    trace = b.cs_trace_collect()
    b.cs_trace_only(None)
    # every kernel's duration, from steps with all launches traced (after the timed ones)
    b.cs_trace_reset()
    for _ in range(breakdown_steps):
        restore()
        torch.cuda.synchronize()
        busy_gpu(torch)
        b.cs_trace_enable(True)
        run_compose(inp, w, rho, b, torch, out, lse, sel, scores, ws, batched, fused, paged)
        b.cs_trace_enable(False)
        torch.cuda.synchronize()
    breakdown = b.cs_trace_collect() if breakdown_steps else None
    # The same steps without the per-kernel trace, whose events cost the host ~14 us per launch: where
    # a layer call's GPU work is short (the 8k-token cache), the traced steps wait on the host.
    untraced = []
    for _ in range(untraced_steps):
        restore()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        busy_gpu(torch)
        e0.record(stream)
        run_compose(inp, w, rho, b, torch, out, lse, sel, scores, ws, batched, fused, paged)
        e1.record(stream)
        torch.cuda.synchronize()
        untraced.append(e0.elapsed_time(e1))
    # algorithmic work of the step (from the selection of the last step; outside the timed region)
    g = sel[:k].cpu().numpy().astype(np.int64)
    visible = int(np.sum(g + 1))
    attn_flops_per_layer = 4 * w.head_dim * w.n_q_heads * visible     # QK^T + PV, 2 flops per MAC
    off = inp.offsets
    cs = w.chunk_start
    rot_tokens = int(sum(cs[c + 1] - cs[c] for c in range(w.n_chunks) if np.any(off[c])))
    rebase_bytes = 2 * w.n_layers * w.n_kv_heads * rot_tokens * w.head_dim * 2   # read + write, bf16
    res = dict(rho=rho, n_sel=k, ms=float(np.median(times)), ms_mean=float(np.mean(times)),
               ms_min=float(np.min(times)), wall_s=wall, steps=steps, trace=trace,
               attn_flops_per_layer=attn_flops_per_layer, rebase_bytes=rebase_bytes, visible=visible,
               ms_untraced=float(np.median(untraced)) if untraced else None,
               breakdown=breakdown, breakdown_steps=breakdown_steps)
    log(f"[bench] rho={rho}: compose median {res['ms']:.3f} ms (min {res['ms_min']:.3f})"
        + (f", untraced {res['ms_untraced']:.3f} ms" if untraced else "") + "; kernels:")
    for name, (cnt, tot) in sorted(trace.items(), key=lambda kv: -kv[1][1]):
        log(f"    {name:24s} launches {cnt:5d}  avg {tot / cnt * 1e3:9.1f} us  total/step {tot / steps:8.3f} ms")
    if breakdown:
        log(f"[bench] rho={rho}: every kernel, {breakdown_steps} more steps with all launches traced:")
        for name, (cnt, tot) in sorted(breakdown.items(), key=lambda kv: -kv[1][1]):
            log(f"    {name:24s} launches {cnt:5d}  avg {tot / cnt * 1e3:9.1f} us  "
                f"total/step {tot / breakdown_steps:8.3f} ms")
    return res


def bench_graph(inp, w, rho, steps, binding, torch):
    """The per-layer composition captured once into a HIP graph and replayed:
    the same kernels, launched by the graph instead of the host.  Caches are
    restored by eager copies before every replay (untimed), and every replay
    is checked bit-identical to an eager composition."""
    b = binding
    n = w.n_candidates
    scores = torch.empty(n, dtype=torch.float32, device="cuda")
    sel = torch.empty(n, dtype=torch.int32, device="cuda")
    k = b.score_deviation_topk(inp.geo, inp.K, w.score_layer, inp.KF[w.score_layer], rho, scores, sel)
    out = torch.empty((w.n_layers, w.n_q_heads, k, w.head_dim), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((w.n_layers, w.n_q_heads, k), dtype=torch.float32, device="cuda")
    ws = torch.empty(max(b.selective_attend_scatter_workspace(inp.geo, k, 1), 1), dtype=torch.uint8, device="cuda")

    def restore():
        inp.K.copy_(inp.K0)
        inp.V.copy_(inp.V0)

    restore()
    run_compose(inp, w, rho, b, torch, out, lse, sel, scores, ws, False)
    torch.cuda.synchronize()
    ref = [t.clone() for t in (inp.K, inp.V, out, lse)]
    restore()
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        run_compose(inp, w, rho, b, torch, out, lse, sel, scores, ws, False)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    times, identical = [], True
    for _ in range(steps + 1):   # the first replay is a warm-up
        restore()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        busy_gpu(torch)
        e0.record(stream)
        graph.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1))
        identical = identical and all(torch.equal(x, y) for x, y in zip((inp.K, inp.V, out, lse), ref))
    del graph
    ms = float(np.median(times[1:]))
    log(f"[bench] rho={rho}: graph-replayed compose median {ms:.3f} ms, replays identical: {identical}")
    return dict(ms=ms, identical=identical)


def _events(torch, stream, fn, reps, before=None):
    """Median milliseconds of fn() between HIP events on the library's stream."""
    times = []
    for _ in range(reps):
        if before is not None:
            before()
        torch.cuda.synchronize()
        busy_gpu(torch)
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        fn()
        e1.record(stream)
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1))
    return float(np.median(times)), float(np.min(times))


def sweep_rebase(args, b, synth, torch):
    """compose_rebase_k on K caches of 8k, 65k and 262k tokens (2048-token chunks, every chunk moved
    on all three axes), restored before every repetition; with a flush, 1 GiB of unrelated data is
    written between the restore and the timed call so that no part of K is still in the caches."""
    stream = torch.cuda.current_stream()
    junk = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    rows = []
    for name in ("rebase8k", "rebase65k", "rebase262k"):
        w = synth.WORKLOADS[name]
        geo = b.Geo.from_workload(w)
        off = synth.chunk_offsets(w)
        K0 = torch.empty((w.n_layers, w.n_kv_heads, w.n_tokens, w.head_dim), dtype=torch.bfloat16, device="cuda")
        for layer in range(w.n_layers):
            K0[layer] = synth.torch_normal((w.n_kv_heads, w.n_tokens, w.head_dim), w.seed, 0, synth.TAG_K, layer,
                                           "cuda", torch.bfloat16)
        K = K0.clone()
        cs = w.chunk_start
        rot = int(sum(cs[c + 1] - cs[c] for c in range(w.n_chunks) if np.any(off[c])))
        nbytes = 2 * w.n_layers * w.n_kv_heads * rot * w.head_dim * 2
        for flush in (True, False):
            def before(flush=flush):
                K.copy_(K0)
                if flush:
                    junk.fill_(7)
            med, best = _events(torch, stream, lambda: b.compose_rebase_k(geo, K, off), args.steps + 1, before)
            gbps = nbytes / (med * 1e-3) / 1e9
            rows.append({"workload": name, "tokens": w.n_tokens, "bytes": nbytes, "flush": flush,
                         "ms": round(med, 4), "ms_min": round(best, 4), "GBps": round(gbps, 1),
                         "frac_hbm": round(gbps / HBM_PEAK_GBPS, 4)})
            log(f"[bench] {name} flush={flush}: {med * 1e3:.1f} us, {gbps:.1f} GB/s")
        del K0, K
    # per-token offsets: scalar re-basing (token j of the composed cache to (j, j, j)) of the
    # 65k-token cache geometry, through compose_rebase_k_tokens
    w = synth.WORKLOADS["long65k"]
    geo = b.Geo.from_workload(w)
    loc = synth.local_coords(w).astype(np.int64)
    j = np.arange(w.n_tokens, dtype=np.int64)
    toff_h = np.stack([j, j, j], axis=1) - loc
    toff = torch.from_numpy(toff_h.astype(np.int32)).cuda()
    moved = int(np.sum(np.any(toff_h != 0, axis=1)))
    nbytes = 2 * w.n_layers * w.n_kv_heads * moved * w.head_dim * 2
    K0 = torch.empty((w.n_layers, w.n_kv_heads, w.n_tokens, w.head_dim), dtype=torch.bfloat16, device="cuda")
    for layer in range(w.n_layers):
        K0[layer] = synth.torch_normal((w.n_kv_heads, w.n_tokens, w.head_dim), w.seed, 0, synth.TAG_K, layer,
                                       "cuda", torch.bfloat16)
    K = K0.clone()
    for flush in (True, False):
        def before(flush=flush):
            K.copy_(K0)
            if flush:
                junk.fill_(7)
        med, best = _events(torch, stream, lambda: b.compose_rebase_k_tokens(geo, K, toff), args.steps + 1, before)
        gbps = nbytes / (med * 1e-3) / 1e9
        rows.append({"workload": "long65k, per-token scalar offsets", "tokens": w.n_tokens, "bytes": nbytes,
                     "flush": flush, "ms": round(med, 4), "ms_min": round(best, 4), "GBps": round(gbps, 1),
                     "frac_hbm": round(gbps / HBM_PEAK_GBPS, 4)})
        log(f"[bench] long65k scalar per-token flush={flush}: {med * 1e3:.1f} us, {gbps:.1f} GB/s")
    # the same cache held as one buffer per chunk (the paged calls), per-chunk and per-token offsets
    cs = w.chunk_start
    Kc0 = [K0[:, :, cs[c]:cs[c + 1]].clone() for c in range(w.n_chunks)]
    Kc = [x.clone() for x in Kc0]
    del K0, K
    off = synth.chunk_offsets(w)
    rot = int(sum(cs[c + 1] - cs[c] for c in range(w.n_chunks) if np.any(off[c])))
    for label, fn, nb in (
            ("long65k paged, per-chunk offsets", lambda: b.compose_rebase_k_paged(geo, Kc, off),
             2 * w.n_layers * w.n_kv_heads * rot * w.head_dim * 2),
            ("long65k paged, per-token scalar offsets", lambda: b.compose_rebase_k_tokens_paged(geo, Kc, toff),
             nbytes)):
        for flush in (True, False):
            def before(flush=flush):
                for x, x0 in zip(Kc, Kc0):
                    x.copy_(x0)
                if flush:
                    junk.fill_(7)
            med, best = _events(torch, stream, fn, args.steps + 1, before)
            gbps = nb / (med * 1e-3) / 1e9
            rows.append({"workload": label, "tokens": w.n_tokens, "bytes": nb, "flush": flush, "ms": round(med, 4),
                         "ms_min": round(best, 4), "GBps": round(gbps, 1), "frac_hbm": round(gbps / HBM_PEAK_GBPS, 4)})
            log(f"[bench] {label} flush={flush}: {med * 1e3:.1f} us, {gbps:.1f} GB/s")
    del Kc, Kc0
    print(json.dumps({"metric": "rebase GB/s (% HBM peak) by cache size", "unit": "GB/s", "n_gpus": 1,
                      "higher_is_better": True, "dtype": "bf16", "data": "synthetic", "sweep": rows}), flush=True)


def sweep_attention(args, b, synth, torch):
    """The 32k-token cache (16 chunks of 2048, 36 layers): one per-layer scatter + attention call at
    each rho; TFLOP/s from the algorithmic flops of the selection over the whole stage's kernels."""
    w = synth.WORKLOADS["attn32k"]
    inp = Inputs(w, torch, b, synth)
    n = w.n_candidates
    stream = torch.cuda.current_stream()
    rows = []
    base = None
    for rho in (1.0, 0.5, 0.2, 0.1, 0.05):
        inp.K.copy_(inp.K0)  # fresh composition: the selection ranks unscattered rows
        inp.V.copy_(inp.V0)
        b.compose_rebase_k(inp.geo, inp.K, inp.offsets)
        scores = torch.empty(n, dtype=torch.float32, device="cuda")
        sel = torch.empty(n, dtype=torch.int32, device="cuda")
        k = b.score_deviation_topk(inp.geo, inp.K, w.score_layer, inp.KF[w.score_layer], rho, scores, sel)
        out = torch.empty((w.n_layers, w.n_q_heads, k, w.head_dim), dtype=torch.bfloat16, device="cuda")
        ws = torch.empty(max(b.selective_attend_scatter_workspace(inp.geo, k, 1), 1), dtype=torch.uint8,
                         device="cuda")
        g = sel[:k].cpu().numpy().astype(np.int64)
        flops = 4 * w.head_dim * w.n_q_heads * int(np.sum(g + 1))   # per layer

        def stage():
            for layer in range(w.n_layers):
                b.selective_attend_scatter(inp.geo, inp.K, inp.V, layer, layer + 1, sel, k, inp.QF, inp.KF,
                                           inp.VF, out, None, ws)
        stage()  # warm-up
        b.cs_trace_reset()
        b.cs_trace_only(("sel_attn_mfma",))  # (the other launches untraced: their events cost GPU time)
        b.cs_trace_enable(True)
        med, _ = _events(torch, stream, stage, max(args.steps // 2, 2))
        b.cs_trace_enable(False)
        b.cs_trace_only(None)
        tr = b.cs_trace_collect()
        an, ams = tr.get("sel_attn_mfma", (1, 0.0))
        kern_tflops = flops / (ams / an * 1e-3) / 1e12
        stage_tflops = w.n_layers * flops / (med * 1e-3) / 1e12
        if base is None:
            base = med
        rows.append({"rho": rho, "n_sel": k, "stage_ms": round(med, 3), "flops_per_layer": flops,
                     "stage_TFLOPs": round(stage_tflops, 1), "kernel_TFLOPs": round(kern_tflops, 1),
                     "kernel_frac_mfma": round(kern_tflops / MFMA_BF16_PEAK_TFLOPS, 4),
                     "speedup_vs_rho1": round(base / med, 3)})
        log(f"[bench] attn32k rho={rho}: k={k}, stage {med:.3f} ms, kernel {kern_tflops:.1f} TFLOP/s")
    print(json.dumps({"metric": "selective attention TFLOP/s (% MFMA peak) by rho, 32k-token cache",
                      "unit": "TFLOP/s", "n_gpus": 1, "higher_is_better": True, "dtype": "bf16",
                      "data": "synthetic", "sweep": rows}), flush=True)


def cpu_baseline(w, rho):
    """The CPU oracle, as it stands, on a bounded sample of the same workload:
    re-basing and attention of ONE of the 36 layers (the scoring layer) plus the
    full score and selection, extrapolated to the 36-layer composition."""
    import oracle
    from paper_2607_19547_amd import synth
    log("[bench] cpu_baseline: building one layer of oracle inputs")
    layer = w.score_layer
    d = oracle.inputs.build(w, layers=[layer])
    th = oracle.rope.inv_freq(w.head_dim, w.base)
    sg = oracle.rope.axis_of_pair(w.sections)
    t0 = time.perf_counter()
    k_reb = oracle.rebase.rebase_stored(d["k_stored"], w.dtype, d["chunk_start"], d["chunk_offsets"], th, sg)
    t_rebase = time.perf_counter() - t0
    t0 = time.perf_counter()
    scores = oracle.score.deviation_f32(oracle.bf16.decode(k_reb[0]), oracle.bf16.decode(d["k_fresh"][0]), w.cs1)
    sel = oracle.select.select_top(scores, oracle.select.n_select(rho, w.n_candidates), w.cs1)
    t_select = time.perf_counter() - t0
    t0 = time.perf_counter()
    kp = oracle.attention.scatter_rows(k_reb[0], d["k_fresh"][0], sel, w.cs1)
    vp = oracle.attention.scatter_rows(d["v_stored"][0], d["v_fresh"][0], sel, w.cs1)
    oracle.attention.attend_rows(oracle.bf16.decode(d["q_fresh"][0]), oracle.bf16.decode(kp),
                                 oracle.bf16.decode(vp), sel, w.cs1)
    t_attn = time.perf_counter() - t0
    total_s = w.n_layers * (t_rebase + t_attn) + t_select
    threads, cpu_model = host_info()
    log(f"[bench] cpu_baseline: rebase/layer {t_rebase:.2f} s, score+select {t_select:.2f} s, "
        f"attention/layer {t_attn:.2f} s -> {total_s:.1f} s per composition (extrapolated)")
    return dict(value=total_s * 1e3, unit="ms", cores=threads, kind="oracle",
                host_cpus=os.cpu_count(), cpu_model=cpu_model,
                sample=(f"1 of {w.n_layers} layers (rebase {t_rebase:.2f} s + scatter/attention "
                        f"{t_attn:.2f} s, measured) x {w.n_layers} + score/select {t_select:.2f} s "
                        f"(measured, full); float64 numpy on the host"))


def _traffic(kernel):
    """HBM bytes per launch from the committed rocprofv3 PMC summary, if it was
    taken on the current kernel source (else None)."""
    path = os.path.join(ROOT, "profiles", "pmc_traffic.json")
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path)).get(kernel)
        src = os.path.join(ROOT, "paper_2607_19547_amd", "csrc", rec["source"])
        if hashlib.sha256(open(src, "rb").read()).hexdigest() != rec["source_sha256"]:
            return None
        return rec["bytes_per_launch"]
    except Exception:
        return None


def emit(args, w, rho, r, rho1, cpu, other=None, fused=None, paged=None, gemm=None, graph=None, load=None):
    tr = r["trace"]
    steps = r["steps"]
    attn_n, attn_ms = tr.get("sel_attn_mfma", (0, 0.0))
    attn_avg_s = attn_ms / max(attn_n, 1) / 1e3
    attn_tflops = r["attn_flops_per_layer"] / attn_avg_s / 1e12 if attn_n else None
    reb_n, reb_ms = tr.get("rebase_bf16_d128", (0, 0.0))
    reb_avg_s = reb_ms / max(reb_n, 1) / 1e3
    reb_gbps = r["rebase_bytes"] / reb_avg_s / 1e9 if reb_n else None
    # every kernel per step: from the fully traced steps when there are (the timed steps trace the
    # roofline kernels only)
    bd, bd_steps = (r["breakdown"], r["breakdown_steps"]) if r.get("breakdown") else (tr, steps)
    # whole attention stage per layer call: scatter (with the plan, in one launch) + attention + combine
    stage = sum(bd.get(k, (0, 0.0))[1] for k in ("plan_scatter", "scatter_rows", "sel_attn_mfma", "sel_attn_combine"))
    stage_tflops = w.n_layers * r["attn_flops_per_layer"] / (stage / bd_steps / 1e3) / 1e12 if stage else None
    line = {
        "metric": "compose ms/65k-token cache; rebase GB/s (% HBM peak); sel-attn TFLOP/s (% MFMA)",
        "value": round(r["ms"], 4),
        "unit": "ms",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(r["ms"], 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": (f"{w.name}: Qwen2.5-VL-3B-shaped bf16 cache, {w.n_layers} layers, "
                                f"{w.n_q_heads}Q/{w.n_kv_heads}KV heads, head_dim {w.head_dim}, "
                                f"{w.n_chunks} chunks x {w.chunk_tokens} = {w.n_tokens} tokens, rho={rho}"),
                   "n_sel": r["n_sel"], "layer_calls": "batched" if args.batched_layers else "per-layer"},
        "rebase_GBps": None if reb_gbps is None else round(reb_gbps, 1),
        "rebase_frac_hbm": None if reb_gbps is None else round(reb_gbps / HBM_PEAK_GBPS, 4),
        "sel_attn_TFLOPs": None if attn_tflops is None else round(attn_tflops, 1),
        "sel_attn_frac_mfma": None if attn_tflops is None else round(attn_tflops / MFMA_BF16_PEAK_TFLOPS, 4),
        "sel_attn_stage_TFLOPs": None if stage_tflops is None else round(stage_tflops, 1),
        "kernels_ms_per_step": {k: round(v[1] / bd_steps, 4) for k, v in bd.items()},
        "roofline": {
            "kernel": "sel_attn_mfma",
            "bound": "mfma",
            "achieved": None if attn_tflops is None else round(attn_tflops, 2),
            "peak": MFMA_BF16_PEAK_TFLOPS,
            "unit": "TFLOP/s",
            "frac": None if attn_tflops is None else round(attn_tflops / MFMA_BF16_PEAK_TFLOPS, 4),
            "traffic": _traffic("sel_attn_mfma"),
            "flops_per_launch": r["attn_flops_per_layer"],
            "avg_launch_us": round(attn_avg_s * 1e6, 2),
        },
        "roofline_rebase": {
            "kernel": "rebase_bf16_d128",
            "bound": "hbm",
            "achieved": None if reb_gbps is None else round(reb_gbps, 1),
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": None if reb_gbps is None else round(reb_gbps / HBM_PEAK_GBPS, 4),
            "traffic": _traffic("rebase_bf16_d128"),
            "bytes_per_launch": r["rebase_bytes"],
            "avg_launch_us": round(reb_avg_s * 1e6, 2),
        },
    }
    if r.get("ms_untraced") is not None:
        line["compose_untraced_ms"] = round(r["ms_untraced"], 4)
    if other is not None:
        line["per_layer_compose_ms" if args.batched_layers else "batched_compose_ms"] = round(other["ms"], 4)
    if fused is not None:
        line["fused_rope_compose_ms"] = round(fused["ms"], 4)
        line["fused_rope_plain_alternating_ms"] = round(fused["plain_ms"], 4)
        for key, name in (("fused_rope_scatter_us_per_layer", "plan_rope_scatter"),
                          ("fused_rope_sel_attn_us", "sel_attn_mfma")):
            fr = fused["trace"].get(name)
            if fr:
                line[key] = round(fr[1] / fr[0] * 1e3, 2)
    if paged is not None:
        line["paged_compose_ms"] = round(paged["ms"], 4)
        pt = paged["trace"]
        for key, name in (("paged_sel_attn_us", "sel_attn_mfma"), ("paged_rebase_us", "rebase_bf16_d128")):
            if name in pt:
                line[key] = round(pt[name][1] / pt[name][0] * 1e3, 2)
    if load is not None:
        line["chunk_load"] = {"bytes": load["bytes"], "copy_ms": round(load["copy"], 3),
                              "load_rebase_ms": round(load["load_rebase"], 3),
                              "copy_then_rebase_ms": round(load["copy_then_rebase"], 3),
                              "pcie_GBps": round(load["bytes"] / load["load_rebase"] / 1e6, 1),
                              "identical": load["identical"]}
    if graph is not None:
        line["graph_compose_ms"] = round(graph["ms"], 4)
        line["graph_replays_identical"] = graph["identical"]
    if rho1 is not None:
        line["rho1_compose_ms"] = round(rho1["ms"], 3)
        line["rho1_over_rho_speedup"] = round(rho1["ms"] / r["ms"], 3)
    if gemm is not None:
        line["context_vendor_gemm_bf16"] = dict(gemm, sel_attn_over_gemm=None if attn_tflops is None
                                                 else round(attn_tflops / gemm["TFLOPs"], 4))
    if cpu is not None:
        line["cpu_baseline"] = cpu
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
