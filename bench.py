"""Decode-attention throughput over the factorized KV cache on one MI355X.

One step = one decode token through every layer: L per-layer dwkv_decode
calls on one stream (the whole hot path: query projection, coefficient and
residual streaming, softmax, value product, split merge).  Inputs are synthetic
and already resident in HBM when the timed region starts.

Prints ONE JSON line on stdout; progress goes to stderr.  Beside the metric
(mean step time, with the median and p10/p90 of the timed steps) it carries
`roofline` (the split-K kernel's achieved bandwidth against the published
peak and against the device's measured read ceiling, with counter traffic
from the committed profile, and the whole step's fraction beside it), `hbm_read_ceiling`, `cpu_baseline` (the
float64 oracle on the host cores) and, unless skipped, the int8-coefficient,
features, probe, append, comparison and control-loop measurements.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0          # MI355X HBM3E, published


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def algorithmic_bytes_per_layer(host) -> list[float]:
    """Bytes one per-layer decode must move: the window's bases, the layer's
    coefficient rows (fp16, or int8 codes with an fp16 scale per 16), the
    window's offsets, the layer's residual indices, codes and scales, the query
    in and the fp32 output out."""
    B, Hk, Hq, d = host.batch, host.n_kv_heads, host.n_q_heads, host.head_dim
    T, rb = host.total_tokens, host.basis_rank
    qbytes = 2
    out = []
    c8 = getattr(host, "coef_format", "f16") == "int8"
    coef_bytes = 2 * Hk * T * (rb + 2 * (rb // 16)) if c8 else 2 * Hk * T * rb * 2
    for l in range(host.n_layers):
        m = l // host.window
        ent = float(host.res_off[m, :, -1].astype(np.int64).sum())      # entries per Z over heads
        out.append(B * Hk * 2 * rb * d * 2          # bases B^K, B^V (fp16)
                   + coef_bytes                     # coefficients A^K, A^V (fp16, or int8 + block scales)
                   + Hk * (T + 1) * 4               # offsets
                   + 2 * ent * 1 + 2 * ent / 2      # channel bytes + int4 codes, K and V
                   + 2 * Hk * T * 2                 # residual scales (fp16), K and V
                   + B * Hq * d * qbytes + B * Hq * d * 4)
    return out


def dense_fp16_bytes_per_layer(host) -> float:
    return 2 * host.n_kv_heads * host.total_tokens * host.head_dim * 2


def cpu_baseline(host, n_pairs: int, budget_s: float):
    """The float64 oracle, as it stands, on a bounded sample of the same step:
    up to n_pairs (layer, KV head) slabs within budget_s seconds, extrapolated
    to the whole step when the sample is not all of it.  `cores` is the thread
    count of the BLAS pool the oracle's numpy runs on (the threads it used),
    `host_cores` the host's logical CPU count."""
    import oracle
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    L, Hk, B = host.n_layers, host.n_kv_heads, host.batch
    pairs = [(l, h) for l in range(L) for h in range(Hk)]
    rng = np.random.default_rng(0)
    n_pairs = len(pairs) if n_pairs <= 0 else min(n_pairs, len(pairs))
    sample = [pairs[i] for i in rng.choice(len(pairs), size=n_pairs, replace=False)]
    t0 = time.perf_counter()
    done = 0
    for l, h in sample:
        oracle.decode(host, l, heads=[(b, h) for b in range(B)])
        done += 1
        if time.perf_counter() - t0 > budget_s:
            break
    dt = time.perf_counter() - t0
    step_s = dt / done * len(pairs)
    return {"value": B / step_s, "unit": "tokens/s", "cores": int(threads), "host_cores": os.cpu_count(),
            "kind": "oracle",
            "sample": (f"all {len(pairs)} (layer, KV head) slabs of one decode step, {dt:.1f} s"
                       if done == len(pairs) else
                       f"{done} of {len(pairs)} (layer, KV head) slabs of one decode step, "
                       f"{dt:.1f} s, extrapolated to the full step ({step_s:.1f} s)")}


def measure_append(dc, host, wl, torch, reps: int = 20):
    """The append/compress path at this workload: one decode token routed in
    every window (dwkv_route_range over [T-1, T)) and compressed in every layer
    (dwkv_compress per layer), replayed as a captured graph so the figure is
    GPU time; and a whole-layer compress of all T tokens (the prefill side).
    Writes into the cache, so it runs after the decode timing."""
    from synth import router_inputs
    T, Hk, d, L = host.total_tokens, host.n_kv_heads, host.head_dim, host.n_layers
    phi, u, theta = router_inputs(wl, host.n_windows, T)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    phi_d, u_d, th_d = dev(phi), dev(u), dev(theta)
    g = torch.Generator(device="cuda").manual_seed(1)
    x1 = [(torch.randn((1, Hk, d), generator=g, device="cuda").half(),
           torch.randn((1, Hk, d), generator=g, device="cuda").half()) for _ in range(L)]

    def append_step():
        dc.route_range(phi_d, u_d, th_d, T - 1, T)
        for l in range(L):
            dc.compress(l, x1[l][0], x1[l][1], T - 1, T)

    out = torch.empty((host.batch, host.n_q_heads, d), dtype=torch.float32, device="cuda")

    def decode_step():
        for l in range(L):
            dc.decode(l, out=out)

    def two_step():                       # append, then decode, layer by layer
        dc.route_range(phi_d, u_d, th_d, T - 1, T)
        for l in range(L):
            dc.compress(l, x1[l][0], x1[l][1], T - 1, T)
            dc.decode(l, out=out)

    def fused_step():                     # the decode that appends, layer by layer
        dc.route_range(phi_d, u_d, th_d, T - 1, T)
        for l in range(L):
            dc.decode_append(l, x1[l][0].view(1, Hk, d), x1[l][1].view(1, Hk, d), out=out)

    stream = torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]

    def graph_us(fn):
        fn()
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            fn()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        ev[0].record(stream)
        for _ in range(reps):
            graph.replay()
        ev[1].record(stream)
        torch.cuda.synchronize()
        t = ev[0].elapsed_time(ev[1]) / reps * 1e3
        del graph
        return t

    step_us = graph_us(append_step)
    dec_us = graph_us(decode_step)
    two_us = graph_us(two_step)
    fused_us = graph_us(fused_step)
    # prefill side: every token of one layer
    xk = torch.randn((T, Hk, d), generator=g, device="cuda").half()
    xv = torch.randn((T, Hk, d), generator=g, device="cuda").half()
    dc.compress(0, xk, xv, 0, T)
    torch.cuda.synchronize()
    n_rep = 3
    ev[0].record(stream)
    for _ in range(n_rep):
        dc.compress(0, xk, xv, 0, T)
    ev[1].record(stream)
    torch.cuda.synchronize()
    layer_ms = ev[0].elapsed_time(ev[1]) / n_rep
    return {"decode_token_append_us_per_step": round(step_us, 2),
            "append_launches_per_step": 3 + L,
            "decode_step_us": round(dec_us, 2),
            "append_then_decode_step_us": round(two_us, 2),
            "decode_append_step_us": round(fused_us, 2),
            "decode_append_overhead_us_per_step": round(fused_us - dec_us, 2),
            "decode_append_launches_per_layer": dc.decode_append_launches,
            "prefill_compress_ms_per_layer": round(layer_ms, 4),
            "prefill_compress_vectors_per_s": round(2 * Hk * T / (layer_ms / 1e3), 1),
            "note": "graph replays: route_range of the new token in every window plus one dwkv_compress per "
                    "layer (append alone); the 32-layer decode alone; route_range then per layer "
                    "dwkv_compress + dwkv_decode; route_range then per layer dwkv_decode_append (the new "
                    "token compressed inside the decode launch); overhead = that minus the decode alone. "
                    "prefill = dwkv_compress of all T tokens of one layer, K and V"}


def measure_int8(wl, torch, steps: int = 20, warmup: int = 5):
    """The same workload with the paper's 8-bit blockwise coefficient form
    (int8 codes, one fp16 scale per token and 16 coefficients): tokens/s of the
    32-layer step and the split-K kernel's achieved bandwidth on its own bytes."""
    from paper_2607_06523_amd import DeviceCache
    from synth import generate
    host = generate(wl.with_(coef_format="int8", name=wl.name + "-int8"))
    dc = DeviceCache(host)
    L = host.n_layers
    stream = torch.cuda.current_stream()
    ws = dc.workspace()
    ws_layer = [dc.new_workspace() for _ in range(L)]
    outs = [torch.empty((host.batch, host.n_q_heads, host.head_dim), dtype=torch.float32, device="cuda")
            for _ in range(L)]
    for _ in range(warmup):
        for l in range(L):
            dc.decode(l, out=outs[l], workspace=ws)
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(5)]
    ev[0].record(stream)
    for _ in range(steps):
        for l in range(L):
            dc.decode(l, out=outs[l], workspace=ws)
    ev[1].record(stream)
    for l in range(L):
        dc.decode_partials(l, workspace=ws_layer[l])
    ev[2].record(stream)
    for l in range(L):
        dc.decode_merge(l, out=outs[l], workspace=ws_layer[l])
    ev[3].record(stream)
    torch.cuda.synchronize()
    ms = ev[0].elapsed_time(ev[1]) / steps
    split_ms = ev[1].elapsed_time(ev[2]) / L
    bl = float(np.mean(algorithmic_bytes_per_layer(host)))
    achieved = bl / (split_ms / 1e3) / 1e9
    res = {"tokens_per_s": round(host.batch / (ms / 1e3), 2), "ms_per_step": round(ms, 4),
           "split_kernel_ms": round(split_ms, 5), "merge_kernel_ms": round(ev[2].elapsed_time(ev[3]) / L, 5),
           "bytes_per_layer_call": int(bl), "achieved_gbps": round(achieved, 1),
           "frac": round(achieved / HBM_PEAK_GBPS, 4),
           "compression_vs_fp16": round(dense_fp16_bytes_per_layer(host) / bl, 3),
           "note": "coefficients in the 8-bit blockwise form: int8 codes, one fp16 scale per token and 16 "
                   "coefficients (tl_kernel int8 variant)"}
    del dc, host
    return res


def measure_features(dc, host, torch, outs, steps: int = 5):
    """A decode step that also emits the router's attention features
    (dwkv_decode_features per layer: the scores-storing split pass, the merge
    and the normalizing features launch), against the plain decode step."""
    import ctypes
    L = host.n_layers
    phi = torch.zeros((host.n_windows, host.n_kv_heads, host.total_tokens, 4), dtype=torch.float32, device="cuda")
    ws = torch.empty(int(dc.lib.dwkv_features_workspace_bytes(ctypes.byref(dc.dims))), dtype=torch.uint8,
                     device="cuda")
    stream = torch.cuda.current_stream()

    def step():
        for l in range(L):
            dc.decode_features(l, phi, out=outs[l], workspace=ws)

    step()
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    ev[0].record(stream)
    for _ in range(steps):
        step()
    ev[1].record(stream)
    torch.cuda.synchronize()
    ms = ev[0].elapsed_time(ev[1]) / steps
    return {"tokens_per_s": round(host.batch / (ms / 1e3), 2), "ms_per_step": round(ms, 4),
            "launches_per_layer": 3,
            "note": "dwkv_decode_features per layer: decode plus per-token attention mass and spike folded "
                    "into the window's router features"}


def measure_control(dc, host, wl, torch, reps: int = 3):
    """The control steps at this workload: budget-driven routing of every
    window and head over all T tokens (two levels: the workload's lowest and
    highest), and the sketch initialization of one window's bases from a
    synthetic prefill.  Both write into the cache, so this runs last."""
    import ctypes
    from synth import router_inputs
    T, Hk, d, w, rb, M = (host.total_tokens, host.n_kv_heads, host.head_dim, host.window, host.basis_rank,
                          host.n_windows)
    stream = torch.cuda.current_stream()

    def timed(fn, n):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        fn()
        torch.cuda.synchronize()
        ev[0].record(stream)
        for _ in range(n):
            fn()
        ev[1].record(stream)
        torch.cuda.synchronize()
        return ev[0].elapsed_time(ev[1]) / n

    res = {}
    two = DeviceCache2(dc, (host.levels[0], host.levels[-1]))
    phi, u, _ = router_inputs(wl, M, T)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    phi_d, u_d = dev(phi), dev(u)
    entries = torch.full((M, Hk), T * host.levels[-1] // 10, dtype=torch.int64, device="cuda")
    codes = torch.empty((M, Hk, T), dtype=torch.uint8, device="cuda")
    offs = torch.empty((M, Hk, T + 1), dtype=torch.int32, device="cuda")
    res["route_budget_ms"] = round(timed(lambda: two.route_budget(phi_d, u_d, entries, 0, T, codes, offs), reps), 4)
    g = torch.Generator(device="cuda").manual_seed(3)
    x = torch.randn((w, 2, T, Hk, d), generator=g, device="cuda", dtype=torch.float16)
    omega = torch.randn((w * T, rb), generator=g, device="cuda", dtype=torch.float16)
    res["sketch_basis_ms_per_window"] = round(timed(lambda: dc.sketch_basis(0, 0, x, omega), reps), 4)
    res["note"] = ("route_budget: all windows and heads over T tokens (levels {lo, hi}); sketch: one window, "
                   "w x T prefill rows per head and Z")
    del x, omega
    return res


class DeviceCache2:
    """The same device cache seen with a two-level table (for budget routing)."""
    def __init__(self, dc, levels):
        from paper_2607_06523_amd import binding
        self.dc = dc
        self.dims, self._keep = binding.make_dims(
            batch=dc.batch, n_layers=dc.n_layers, window=dc.window, n_kv_heads=dc.n_kv_heads,
            n_q_heads=dc.n_q_heads, head_dim=dc.head_dim, basis_rank=dc.basis_rank, levels=tuple(levels),
            cu_seqlens_host=dc.cu_host, cu_seqlens_dev_ptr=dc.cu.data_ptr(), total_tokens=dc.total_tokens,
            res_stride=dc.res_stride, split_tokens=0)

    def route_budget(self, phi, u, entries, t0, t1, codes, offs):
        import ctypes
        from paper_2607_06523_amd import binding
        lib, torch = self.dc.lib, self.dc.torch
        need = int(lib.dwkv_route_budget_workspace_bytes(ctypes.byref(self.dims)))
        ws = getattr(self, "_ws", None)
        if ws is None or ws.numel() < need:
            ws = self._ws = torch.empty(need, dtype=torch.uint8, device="cuda")
        p = lambda t: ctypes.c_void_p(t.data_ptr())
        st = lib.dwkv_route_budget(ctypes.byref(self.dims), p(phi), p(u), p(entries), int(t0), int(t1), p(codes),
                                   p(offs), p(ws), ws.numel(), ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
        binding.check(st, "dwkv_route_budget")


def measure_probe(dc, host, torch, steps: int = 5, warmup: int = 2):
    """The decode step with the Eq. 3 probe on one KV head and on all of them:
    each layer runs the factorized decode plus the dense reference pass over
    the probed heads' fp16 reference cache and the probe error.  Every layer
    has its own synthetic reference (random fp16, all T tokens), so no layer
    finds another's reference in a cache."""
    from paper_2607_06523_amd import ProbeRef
    L, T, d, Hk = host.n_layers, host.total_tokens, host.head_dim, host.n_kv_heads
    T16 = -(-T // 16) * 16
    stream = torch.cuda.current_stream()
    res = {}
    for heads in ((0,), tuple(range(Hk))):
        n = len(heads)
        gen = torch.Generator(device="cuda").manual_seed(7)
        probes = [ProbeRef(list(heads), torch.randn((n, T, d), device="cuda", generator=gen).half(),
                           torch.randn((n, T16 // 16, d, 16), device="cuda", generator=gen).half())
                  for _ in range(L)]
        ws = dc.new_workspace(probes[0])

        def step():
            for l in range(L):
                dc.decode(l, probe=probes[l], workspace=ws)
        for _ in range(warmup):
            step()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        torch.cuda.synchronize()
        ev[0].record(stream)
        for _ in range(steps):
            step()
        ev[1].record(stream)
        torch.cuda.synchronize()
        ms = ev[0].elapsed_time(ev[1]) / steps
        res[f"probe_{n}_heads"] = {"tokens_per_s": round(host.batch / (ms / 1e3), 2), "ms_per_step": round(ms, 4),
                                   "reference_bytes_per_layer": int(n * T * d * 2 * 2)}
        del probes, ws
    res["note"] = ("dwkv_decode with a probe on every layer (each layer its own fp16 reference): the factorized "
                   "decode plus a dense split pass over the probed heads' reference and the Eq. 3 error in the "
                   "merge")
    return res


def measure_comparators(dc, host, torch, steps: int = 3):
    """The decode's comparison paths on the same GPU and workload: a dense fp16
    cache decode (every layer's K/V resident, 2 bytes per element) and the
    unfused path (each layer's cache rebuilt into fp16 buffers, then the dense
    decode over them).  Times whole 32-layer steps with HIP events, plus the
    per-layer kernels."""
    T, Hk, d, L, B = host.total_tokens, host.n_kv_heads, host.head_dim, host.n_layers, host.batch
    T16 = -(-T // 16) * 16
    g = torch.Generator(device="cuda").manual_seed(2)
    ks = [torch.randn((Hk, T, d), generator=g, device="cuda", dtype=torch.float16) for _ in range(L)]
    vs = [torch.randn((Hk, T16 // 16, d, 16), generator=g, device="cuda", dtype=torch.float16) for _ in range(L)]
    kb = torch.empty((Hk, T, d), dtype=torch.float16, device="cuda")
    vb = torch.empty((Hk, T16 // 16, d, 16), dtype=torch.float16, device="cuda")
    outs = [torch.empty((B, host.n_q_heads, d), dtype=torch.float32, device="cuda") for _ in range(L)]
    ws = torch.empty(int(dc.lib.dwkv_dense_workspace_bytes(__import__("ctypes").byref(dc.dims))),
                     dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()

    def timed(fn, n):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        fn()
        torch.cuda.synchronize()
        ev[0].record(stream)
        for _ in range(n):
            fn()
        ev[1].record(stream)
        torch.cuda.synchronize()
        return ev[0].elapsed_time(ev[1]) / n

    dense_step = timed(lambda: [dc.dense_decode(ks[l], vs[l], dc.q[l], out=outs[l], workspace=ws)
                                for l in range(L)], steps)
    unfused_step = timed(lambda: [(dc.materialize(l, kb, vb), dc.dense_decode(kb, vb, dc.q[l], out=outs[l],
                                                                              workspace=ws))
                                  for l in range(L)], steps)
    mat_layer = timed(lambda: [dc.materialize(l, kb, vb) for l in range(L)], steps) / L
    dense_bytes = 2 * Hk * T * d * 2 + B * host.n_q_heads * d * (2 + 4)
    dense_layer = dense_step / L
    del ks, vs
    return {"dense_fp16_tokens_per_s": round(B / (dense_step / 1e3), 2),
            "dense_fp16_ms_per_step": round(dense_step, 4),
            "dense_fp16_gbps": round(dense_bytes / (dense_layer / 1e3) / 1e9, 1),
            "unfused_tokens_per_s": round(B / (unfused_step / 1e3), 2),
            "unfused_ms_per_step": round(unfused_step, 4),
            "materialize_ms_per_layer": round(mat_layer, 5),
            "note": "dense: dwkv_dense_decode per layer over resident fp16 K/V; unfused: dwkv_materialize "
                    "then dwkv_dense_decode per layer (rebuilt cache written to and re-read from HBM)"}


def measure_hbm_ceiling(torch, gib: int = 4, reps: int = 10):
    """Practical HBM read ceiling: dwkv_hbm_read over a buffer far beyond the
    last-level caches, timed with HIP events on the current stream."""
    from paper_2607_06523_amd import hbm_read, hbm_read_blocks
    buf = torch.ones(gib << 28, dtype=torch.int32, device="cuda")
    sink = torch.empty(hbm_read_blocks(), dtype=torch.int32, device="cuda")
    for _ in range(3):
        hbm_read(buf, sink)
    stream = torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    ev[0].record(stream)
    for _ in range(reps):
        hbm_read(buf, sink)
    ev[1].record(stream)
    torch.cuda.synchronize()
    ms = ev[0].elapsed_time(ev[1]) / reps
    nbytes = buf.numel() * 4
    del buf, sink
    return {"gbps": round(nbytes / (ms / 1e3) / 1e9, 1), "bytes": nbytes, "ms": round(ms, 4), "reps": reps,
            "kernel": "stream_read_kernel (dwkv_hbm_read): 1 KB nontemporal loads per wave instruction"}


def measured_traffic(workload: str):
    """HBM bytes per launch of the token-lane decode kernel from the committed
    rocprofv3 counter profile, or None when that profile is missing or was
    taken on a different kernel source."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"tl_kernel_{workload}_hbm_bytes.json")
    src = os.path.join(ROOT, "paper_2607_06523_amd", "csrc", "decode_tl.hip")
    try:
        rec = json.load(open(path))
        sha = hashlib.sha256(open(src, "rb").read()).hexdigest()
    except (OSError, ValueError):
        return None
    if rec.get("kernel_source_sha256") != sha:
        return None
    return float(rec["traffic_bytes_per_launch"])


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="llama8b-64k")
    ap.add_argument("--context", type=int, default=0,
                    help="override the workload's context length in tokens (same shape otherwise)")
    ap.add_argument("--split", type=int, default=0, help="tokens per workgroup chunk (0 = automatic)")
    ap.add_argument("--variant", default="full", choices=["full", "bases-only"],
                    help="bases-only: every routed residual rank 0 (shared bases only)")
    ap.add_argument("--graph", action="store_true", help="replay the step as a captured HIP graph")
    ap.add_argument("--coef", default="fp16", choices=["fp16", "int8"],
                    help="coefficient format of the timed workload (int8: the 8-bit blockwise form)")
    ap.add_argument("--probe-heads", type=int, default=-1,
                    help="KV heads probed (Eq. 3) in every layer of the timed step, each layer with its own "
                         "fp16 reference; -1 = the workload's setting (one head when it probes every layer)")
    ap.add_argument("--cpu-pairs", type=int, default=0, help="slabs to time on the CPU (0 = all)")
    ap.add_argument("--cpu-budget", type=float, default=20.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-append", action="store_true", help="skip the append/compress measurement")
    ap.add_argument("--no-comparators", action="store_true",
                    help="skip the dense fp16 and unfused comparison paths")
    ap.add_argument("--copy-calib-mib", type=int, default=0,
                    help="before timing, run one plain device copy of this many MiB (a known-size "
                         "reference for HBM byte counters)")
    ap.add_argument("--hbm-ceiling-only", action="store_true",
                    help="only time the HBM read stream (dwkv_hbm_read) and print its JSON")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              f"(the decode path shards by KV head across GPUs with no exchange, see the design notes)",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2607_06523_amd import DeviceCache, binding
    if not os.path.exists(binding.LIB_PATH):
        from paper_2607_06523_amd.build import build
        build()
    if args.hbm_ceiling_only:
        print(json.dumps({"hbm_read_ceiling": measure_hbm_ceiling(torch)}), flush=True)
        return
    from synth import ALL, generate

    wl = ALL[args.workload]
    if args.context > 0 and args.context != wl.context:
        wl = wl.with_(context=args.context, name=f"{wl.name.rsplit('-', 1)[0]}-{args.context // 1024}k")
    if args.variant == "bases-only":
        wl = wl.with_(levels=(0,), probs=(1.0,), salient_frac=0.0, name=wl.name + "-bases-only")
    if args.coef == "int8":
        wl = wl.with_(coef_format="int8", name=wl.name + "-int8")
    log(f"[bench] generating {wl.name} ({wl.description})")
    t = time.time()
    host = generate(wl)
    log(f"[bench] generated in {time.time() - t:.1f} s")
    dc = DeviceCache(host, split_tokens=args.split)
    L = host.n_layers
    stream = torch.cuda.current_stream()
    outs = [torch.empty((host.batch, host.n_q_heads, host.head_dim), dtype=torch.float32, device="cuda")
            for _ in range(L)]
    n_probe = args.probe_heads if args.probe_heads >= 0 else (1 if getattr(wl, "probe", False) else 0)
    probes = errs = None
    if n_probe > 0:
        # one synthetic fp16 reference per layer for the first n_probe KV heads
        from paper_2607_06523_amd import ProbeRef
        T, d = host.total_tokens, host.head_dim
        T16 = -(-T // 16) * 16
        gen = torch.Generator(device="cuda").manual_seed(7)
        probes = [ProbeRef(list(range(n_probe)), torch.randn((n_probe, T, d), device="cuda", generator=gen).half(),
                           torch.randn((n_probe, T16 // 16, d, 16), device="cuda", generator=gen).half())
                  for _ in range(L)]
        errs = [torch.empty((host.batch, n_probe * wl.group), dtype=torch.float32, device="cuda") for _ in range(L)]
        log(f"[bench] probe: {n_probe} KV head(s) in every layer, {len(probes)} references")
    ws = dc.workspace(probes[0] if probes else None)

    def step():
        for l in range(L):
            if probes:
                dc.decode(l, out=outs[l], workspace=ws, probe=probes[l], err=errs[l], with_ref=False)
            else:
                dc.decode(l, out=outs[l], workspace=ws)

    if args.copy_calib_mib > 0:
        n = args.copy_calib_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        log(f"[bench] calibration copy: {args.copy_calib_mib} MiB read + {args.copy_calib_mib} MiB written")

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    graph = None
    if args.graph:
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step()
        torch.cuda.synchronize()
        for _ in range(2):
            graph.replay()
        torch.cuda.synchronize()

    # timed region: K steps.  The last step runs every layer as its two
    # halves: first the split-K pass of all L layers back to back (each layer
    # into its own workspace), then the L merges, with one event pair around
    # each run on the kernels' stream.  That times the split-K kernel (the
    # dominant one) on its own without an event between every pair of launches.
    ev_step = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    ev_calls = [torch.cuda.Event(enable_timing=True) for _ in range(3)] if graph is None else None
    ws_layer = ([dc.new_workspace(probes[0] if probes else None) for _ in range(L)]
                if graph is None else None)
    torch.cuda.synchronize()
    ev_step[0].record(stream)
    wall0 = time.perf_counter()
    for k in range(args.steps):
        if graph is not None:
            graph.replay()
        elif k == args.steps - 1:
            ev_calls[0].record(stream)
            for l in range(L):
                dc.decode_partials(l, workspace=ws_layer[l], probe=probes[l] if probes else None,
                                   err=errs[l] if probes else None)
            ev_calls[1].record(stream)
            for l in range(L):
                dc.decode_merge(l, out=outs[l], workspace=ws_layer[l], probe=probes[l] if probes else None,
                                err=errs[l] if probes else None)
            ev_calls[2].record(stream)
        else:
            step()
        ev_step[k + 1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    total_ms = ev_step[0].elapsed_time(ev_step[args.steps])
    ms_per_step = total_ms / args.steps
    per_step = np.array([ev_step[k].elapsed_time(ev_step[k + 1]) for k in range(args.steps)])
    split_ms = merge_ms = None
    if ev_calls is not None:
        split_ms = ev_calls[0].elapsed_time(ev_calls[1]) / L
        merge_ms = ev_calls[1].elapsed_time(ev_calls[2]) / L

    bytes_layer = algorithmic_bytes_per_layer(host)
    probe_bytes_layer = 0.0
    if probes:       # the dense fp16 reference keys and values of the probed heads, read once per layer
        probe_bytes_layer = float(n_probe * host.total_tokens * host.head_dim * 2 * 2)
        bytes_layer = [b + probe_bytes_layer for b in bytes_layer]
    bytes_step = float(sum(bytes_layer))
    tok_s = host.batch / (ms_per_step / 1e3)
    step_gbps = bytes_step / (ms_per_step / 1e3) / 1e9
    if split_ms is not None:
        avg_split_ms = float(split_ms)
        achieved = float(np.mean(bytes_layer)) / (avg_split_ms / 1e3) / 1e9
    else:
        avg_split_ms = ms_per_step / L
        achieved = step_gbps
    traffic = measured_traffic(wl.name) if args.variant == "full" and args.split == 0 else None
    ceiling = measure_hbm_ceiling(torch)
    result = {
        "metric": "compressed-KV decode attn tokens/s at 64K ctx (plus achieved HBM GB/s)",
        "value": round(tok_s, 2),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "ms_per_step_median": round(float(np.median(per_step)), 4),
        "ms_per_step_p10": round(float(np.percentile(per_step, 10)), 4),
        "ms_per_step_p90": round(float(np.percentile(per_step, 90)), 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic",
        "config": {"workload": wl.name, "variant": args.variant, "batch": host.batch, "context": wl.context,
                   "layers": L, "window": wl.window, "kv_heads": wl.n_kv_heads,
                   "q_heads": wl.n_q_heads, "head_dim": wl.head_dim, "basis_rank": wl.basis_rank,
                   "levels": list(wl.levels), "split_tokens": dc.split_tokens,
                   "graph": bool(graph is not None)},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": traffic,
                     "kernel": ("split-K partials pass (the dominant kernel: "
                                + ("tl_kernel" if dc.uses_token_lane else "split_kernel") + " at this workload)"
                                if not probes else
                                "split-K phase of the probed step: the factorized pass and the probe's dense "
                                "reference pass, over both passes' bytes"),
                     "measured_ceiling": ceiling["gbps"], "frac_of_measured_ceiling": round(achieved / ceiling["gbps"], 4),
                     "whole_step": {"achieved": round(step_gbps, 1), "frac": round(step_gbps / HBM_PEAK_GBPS, 4),
                                    "note": "algorithmic bytes of all L per-layer calls / the whole step's time "
                                            "(split-K pass, merge and launch gaps)"}},
        "hbm_read_ceiling": ceiling,
        "step_gbps": round(step_gbps, 1),
        "bytes_per_step": int(bytes_step),
        "bytes_per_layer_call": int(np.mean(bytes_layer)),
        "launches_per_layer": dc.decode_launches,
        "split_kernel_ms": round(avg_split_ms, 5),
        "merge_kernel_ms": round(float(merge_ms), 5) if merge_ms is not None else None,
        "compression_vs_fp16": round(dense_fp16_bytes_per_layer(host) / (np.mean(bytes_layer) - probe_bytes_layer), 3),
        "probe": ({"kv_heads_per_layer": n_probe, "reference_bytes_per_layer": int(probe_bytes_layer),
                   "note": "Eq. 3 probe in every layer: dense fp16 reference pass of the probed heads plus the "
                           "probe merge; its bytes are included in bytes_per_layer_call and the roofline"}
                  if probes else None),
        "kv_token_layers_per_s": round(host.total_tokens * L / (ms_per_step / 1e3), 1),
        "wall_s_timed": round(wall, 3),
    }
    if not args.no_comparators and args.variant == "full":
        log("[bench] timing the 8-bit blockwise coefficient form")
        result["coef_int8"] = measure_int8(wl, torch)
        log("[bench] timing the decode with router features")
        result["with_features"] = measure_features(dc, host, torch, outs)
    if not args.no_append and args.variant == "full":
        log("[bench] timing the append/compress path")
        result["append"] = measure_append(dc, host, wl, torch)
    if not args.no_comparators and args.variant == "full":
        log("[bench] timing the dense fp16 and unfused comparison paths")
        result["comparators"] = measure_comparators(dc, host, torch)
    if not args.no_comparators and args.variant == "full":
        log("[bench] timing the decode with the Eq. 3 probe")
        result["with_probe"] = measure_probe(dc, host, torch)
    if not args.no_comparators and args.variant == "full":
        log("[bench] timing the control steps (budget routing, sketch bases)")
        result["control"] = measure_control(dc, host, wl, torch)
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a sample")
        result["cpu_baseline"] = cpu_baseline(host, args.cpu_pairs, args.cpu_budget)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
