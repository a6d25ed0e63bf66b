#!/usr/bin/env python3
"""Benchmark of the activation-sparse FFN forward pass at decode on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-sweep] [--no-cpu]

A *step* is one FFN forward call through the C ABI: gate GEMV (standard W_gate x or
LoPA B (A x)), threshold and compaction, gathered W_up dot products, gathered W_down
accumulation.  Weight sets are resident in HBM before timing and rotate every step
(each step also takes a different token), with enough sets that the per-rotation
footprint exceeds the 256 MB Infinity Cache.  K steps are captured in a HIP graph
and replayed once inside the timed region, which is bracketed by device
synchronization; the reported time per call is that wall-clock time / K.

Printed: ONE JSON line for the headline workload (the largest single-GPU shape: the
Llama-3-70B-shaped FFN, d 8192, d_ff 28672, bf16 weights, standard gating, t for 90%
sparsity, T = 1), with

* ``value``            µs per sparse FFN call (lower is better)
* ``speedup_vs_dense`` dense-path time / sparse-path time, same shape and rotation
* ``hbm_gbps_touched`` algorithmic bytes touched per call / time per call (the
                       call-level fraction of peak is ``hbm_frac_touched``)
* ``roofline``         the dominant (gate) kernel alone: algorithmic bytes per launch /
                       its average duration from hipExtLaunchKernel start/stop events
* ``us_per_call_mall_flushed``  the same call eager, each after a 1 GiB write that evicts
                       the Infinity Cache and the L2s (median of 20; also on the sweep's
                       single-token rows)
* ``cpu_baseline``     the fp64 oracle on one host core for a bounded sample of the
                       headline workload (and the dense oracle on three calls)
* ``sweep``            the other workloads (70B LoPA and 8-token batches; 8B standard
                       50/80/90/95%, LoPA 90/95%, batched LoPA, full form, int8 / int4;
                       the tiny fp32 case), each with its own dense baselines, including
                       the dense FFN written with torch bf16 products.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "µs/FFN-call + speedup vs dense at 90% sparsity; HBM GB/s on bytes touched"
PEAK_HBM_GBPS = 8000.0
MALL_BYTES = 256 << 20


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=400)
    ap.add_argument("--warmup", type=int, default=40)
    ap.add_argument("--workload", default="70b_std_s90_T1")
    ap.add_argument("--no-sweep", action="store_true", help="time the headline workload only")
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle CPU baseline")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain 256 MiB device copy (reference for HBM byte counters)")
    return ap.parse_args()


# ---------------------------------------------------------------- weight sets in HBM
class Shape:
    """Weight sets of one FFN shape, resident in HBM: W_up / W_down^T shared by standard
    and LoPA gating, W_gate for standard, (A, B) per LoPA rank.  Set 0 comes from the
    seeded numpy generator (the oracle's inputs); sets 1.. are drawn on the device with
    a seeded torch generator from the same distributions."""

    def __init__(self, d, d_ff, ranks, n_sets, seed, pool, wdt=None):
        import torch
        from paper_2609_31975_amd import workloads as wl
        wdt = wl.BF16 if wdt is None else wdt
        self.d, self.d_ff, self.n_sets, self.seed, self.wdt = d, d_ff, n_sets, seed, wdt
        self.host0 = {r: wl.make_inputs(seed, 1, d, d_ff, r=r, wdt=wdt) for r in ranks}
        h0 = self.host0[ranks[0]]
        self.pool = pool
        self.x = []
        self.up, self.down, self.gate, self.lopa = [], [], [], {r: [] for r in ranks if r}
        # quantized sets: the row scales of each matrix, same indexing as the codes
        self.s_up, self.s_down, self.s_gate, self.s_lopa = [], [], [], {r: [] for r in ranks if r}
        g = torch.Generator(device="cuda")
        quant = wdt in wl.QMAX

        def bf16(a):
            if a.dtype != np.uint16:  # int8 / packed int4 codes, float32 scales
                return torch.from_numpy(a).to("cuda")
            return torch.from_numpy(a.view(np.int16)).to("cuda").view(torch.bfloat16)

        def randn(shape, std, k, tag):
            g.manual_seed(seed * 1000003 + k * 101 + tag)
            if not quant:
                dt = torch.float32 if wdt == wl.F32 else torch.bfloat16
                return (torch.randn(shape, generator=g, device="cuda") * std).to(dt)
            # codes and row scales drawn as the seeded generator does, on the device
            qmax = wl.QMAX[wdt]
            sq = qmax / 3.0
            q = torch.clamp(torch.round(torch.randn(shape, generator=g, device="cuda") * sq), -qmax, qmax)
            q = q.to(torch.int8)
            if wdt == wl.I4:
                q = ((q[:, 0::2].to(torch.uint8) & 15) | ((q[:, 1::2].to(torch.uint8) & 15) << 4)).contiguous()
            sc = (std / sq) * (0.8 + 0.4 * torch.rand(shape[0], generator=g, device="cuda"))
            return q, sc.to(torch.float32)

        def put(codes_list, scale_list, v):
            if quant:
                codes_list.append(v[0])
                scale_list.append(v[1])
            else:
                codes_list.append(v)

        for k in range(n_sets):
            if k == 0:
                self.x.append(torch.from_numpy(wl.make_tokens(seed, pool, d)).to("cuda"))

                def host(h, name, key):
                    a = bf16(getattr(h, name))
                    return (a, bf16(h.scales[key])) if quant else a
                put(self.up, self.s_up, host(h0, "w_up", "up"))
                put(self.down, self.s_down, host(h0, "w_down_t", "down"))
                if 0 in ranks:
                    put(self.gate, self.s_gate, host(self.host0[0], "w_gate", "gate"))
                else:
                    self.gate.append(None)
                for r in self.lopa:
                    a, b = host(self.host0[r], "lopa_a", "a"), host(self.host0[r], "lopa_b", "b")
                    if quant:
                        self.lopa[r].append((a[0], b[0]))
                        self.s_lopa[r].append((a[1], b[1]))
                    else:
                        self.lopa[r].append((a, b))
            else:
                g.manual_seed(seed * 1000003 + k * 101)
                self.x.append(torch.randn((pool, d), generator=g, device="cuda"))
                put(self.up, self.s_up, randn((d_ff, d), d ** -0.5, k, 1))
                put(self.down, self.s_down, randn((d_ff, d), d_ff ** -0.5, k, 2))
                if 0 in ranks:
                    put(self.gate, self.s_gate, randn((d_ff, d), d ** -0.5, k, 3))
                else:
                    self.gate.append(None)
                for r in self.lopa:
                    a, b = randn((r, d), d ** -0.5, k, 4 + 2 * r), randn((d_ff, r), r ** -0.5, k, 5 + 2 * r)
                    if quant:
                        self.lopa[r].append((a[0], b[0]))
                        self.s_lopa[r].append((a[1], b[1]))
                    else:
                        self.lopa[r].append((a, b))
        torch.cuda.synchronize()


# bytes per weight of each format (fp32, bf16, int8, int4); quantized rows add a 4-byte scale
WEIGHT_BYTES = {0: 4, 1: 2, 2: 1, 3: 0.5}


def algorithmic_bytes(d, d_ff, r, T, n_union, dense, wdt=1):
    """Bytes the method must move per call (weights in format wdt, fp32 x and y)."""
    wb, sb = WEIGHT_BYTES[wdt], (4 if wdt >= 2 else 0)
    gate = (wb * (r * d + d_ff * r) + sb * (r + d_ff)) if r else (wb * d * d_ff + sb * d_ff)
    rows = d_ff if dense else n_union
    return gate + 2 * (wb * d + sb) * rows + 8 * T * d


def gate_kernel_bytes(d, d_ff, r, T, n_union, dense, wdt=1):
    """Algorithmic bytes of the gate kernel: the gate matrix (B for LoPA), the W_up rows
    it reads, and the tokens."""
    wb, sb = WEIGHT_BYTES[wdt], (4 if wdt >= 2 else 0)
    gate = (wb * d_ff * r if r else wb * d * d_ff) + sb * d_ff
    rows = d_ff if dense else n_union
    return gate + (wb * d + sb) * rows + 4 * T * d + (4 * T * r if r else 0)


# ---------------------------------------------------------------- timing
class Runner:
    """Enqueues step i of a workload: weight set i % n_sets, token batch (i // n_sets) % batches."""

    def __init__(self, shape: Shape, r, T, t, dense, form=None, rho=0.0):
        import torch
        from paper_2609_31975_amd import ffn
        self.ffn, self.torch = ffn, torch
        self.s, self.r, self.T, self.t, self.dense = shape, r, T, t, dense
        # correlated batches: each batch of T tokens shares a common N(0, 1) part
        self.xc = None
        if rho > 0:
            g = torch.Generator(device="cuda").manual_seed(7919)
            nb = shape.pool // T
            self.xc = []
            for xs in shape.x:
                c = torch.randn((nb, 1, shape.d), generator=g, device="cuda")
                mix = rho ** 0.5 * c + (1.0 - rho) ** 0.5 * xs[:nb * T].view(nb, T, shape.d)
                self.xc.append(mix.reshape(nb * T, shape.d).contiguous())
        # the full form: option arrays on the device, held for the runner's lifetime
        self.form = form
        self.opt = None if form is None else ffn.options(**form)
        self.batches = shape.pool // T
        self.ws = ffn.alloc_workspace(T, shape.d, shape.d_ff, r)
        self.y = torch.empty((T, shape.d), dtype=torch.float32, device="cuda")

    def args(self, i):
        s = self.s
        k = i % s.n_sets
        b = (i // s.n_sets) % self.batches
        pool = s.x if self.xc is None else self.xc
        return k, pool[k][b * self.T:(b + 1) * self.T]

    def __call__(self, i):
        s, f = self.s, self.ffn
        k, x = self.args(i)
        if s.wdt >= 2:  # quantized weights: the _q calls with the set's row scales
            if self.r:
                a, b = s.lopa[self.r][k]
                sa, sb = s.s_lopa[self.r][k]
                sc = f.scales(lopa_a=sa, lopa_b=sb, up=s.s_up[k], down=s.s_down[k])
                fn = f.ffn_lopa_dense_forward_q if self.dense else f.ffn_lopa_sparse_forward_q
                fn(x, a, b, s.up[k], s.down[k], sc, self.t, self.opt, self.y, self.ws)
            else:
                sc = f.scales(gate=s.s_gate[k], up=s.s_up[k], down=s.s_down[k])
                fn = f.ffn_dense_forward_q if self.dense else f.ffn_sparse_forward_q
                fn(x, s.gate[k], s.up[k], s.down[k], sc, self.t, self.opt, self.y, self.ws)
        elif self.opt is not None:
            a, b = s.lopa[self.r][k]
            fn = f.ffn_lopa_dense_forward_ex if self.dense else f.ffn_lopa_sparse_forward_ex
            fn(x, a, b, s.up[k], s.down[k], self.t, self.opt, self.y, self.ws)
        elif self.r:
            a, b = s.lopa[self.r][k]
            fn = f.ffn_lopa_dense_forward if self.dense else f.ffn_lopa_sparse_forward
            fn(x, a, b, s.up[k], s.down[k], self.t, self.y, self.ws)
        else:
            fn = f.ffn_dense_forward if self.dense else f.ffn_sparse_forward
            fn(x, s.gate[k], s.up[k], s.down[k], self.t, self.y, self.ws)

    def union_sizes(self, K, cap=400):
        """Active-union size of every step (eager, synchronizing); steps past `cap` reuse the
        sizes of the first `cap` steps of the rotation."""
        n = {}
        period = min(self.s.n_sets * self.batches, cap)
        for i in range(min(K, period)):
            self(i)
            idx, _ = self.ffn.ffn_active_set(self.ws, self.T, self.s.d, self.s.d_ff, self.r, with_act=False)
            n[i] = len(idx)
        return [n[i % period] for i in range(K)]


def time_graph(run: Runner, K: int, W: int):
    """Warm up W eager steps, capture K steps in a graph, replay once untimed, then time one
    replay between device synchronizations.  Returns µs per step (wall clock and events)."""
    torch = run.torch
    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        for i in range(W):
            run(i)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=stream):
        for i in range(K):
            run(i)
    with torch.cuda.stream(stream):
        graph.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    with torch.cuda.stream(stream):
        torch.cuda.synchronize()
        w0 = time.perf_counter()
        e0.record(stream)
        graph.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        w1 = time.perf_counter()
    del graph
    return (w1 - w0) * 1e6 / K, e0.elapsed_time(e1) * 1e3 / K


FLUSH_BYTES = 1 << 30


def time_flushed(run: Runner, n: int = 20):
    """Median µs of n eager calls, each after a 1 GiB write that evicts the 256 MB Infinity
    Cache and the L2s: its own event pair around the call only.  The host enqueues the call
    while the write runs, so the call's kernels follow one another as in the graph."""
    torch = run.torch
    buf = torch.empty(FLUSH_BYTES, dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
    run(0)
    torch.cuda.synchronize()
    for i, (a, b) in enumerate(evs):
        buf.fill_(i & 0xFF)
        a.record(stream)
        run(i)
        b.record(stream)
    torch.cuda.synchronize()
    del buf
    return float(np.median([a.elapsed_time(b) * 1e3 for a, b in evs]))


def time_gate_kernel(run: Runner, K: int):
    """Average gate-kernel duration over K eager steps (hipExtLaunchKernel start/stop
    events).  A bounded device spin is queued first so that the host enqueues all K
    steps before the GPU reaches them: the kernels then run back to back, as in the
    timed region, instead of on an idle, down-clocked GPU."""
    torch = run.torch
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(K)]
    stream = torch.cuda.current_stream()
    for a, b in evs:  # materialize the event handles
        a.record(stream)
        b.record(stream)
    for i in range(min(K, 8)):
        run(i)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(min(K, 8)):
        run(i)
    per_call_host = (time.perf_counter() - t0) / min(K, 8)
    torch.cuda.synchronize()
    torch.cuda._sleep(int(min(2.0, 1.5 * K * per_call_host + 2e-3) * 2.4e9))
    for i in range(K):
        run.ffn.ffn_time_next_gate_kernel(*evs[i])
        run(i)
    torch.cuda.synchronize()
    d = np.array([a.elapsed_time(b) * 1e3 for a, b in evs])
    return float(d.mean()), float(np.median(d))


def steps_for(run: Runner, K: int, budget_s: float = 1.0) -> int:
    """K, or fewer steps for a slow workload so that its timed region stays near budget_s."""
    torch = run.torch
    run(0)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    run(1)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    return int(max(10, min(K, budget_s / max(dt, 1e-7))))


def measure(shape, r, T, t, K, W, dense_us=None, name="", exact=False, form=None, rho=0.0):
    sp = Runner(shape, r, T, t, dense=False, form=form, rho=rho)
    if not exact:
        K = steps_for(sp, K)
        W = min(W, K)
    n = sp.union_sizes(K)
    us_wall, us_ev = time_graph(sp, K, W)
    nbar = float(np.mean(n))
    by = np.mean([algorithmic_bytes(shape.d, shape.d_ff, r, T, k, False, shape.wdt) for k in n])
    rec = dict(workload=name, gating="lopa" if r else "standard", r=r, T=T, t=t, d=shape.d, d_ff=shape.d_ff,
               weight_sets=shape.n_sets, steps=K, us_per_call=round(us_wall, 3), us_per_call_events=round(us_ev, 3),
               n_union=round(nbar, 1), realized_union_frac=round(nbar / shape.d_ff, 4),
               bytes_per_call=int(by), hbm_gbps_touched=round(by / us_wall / 1e3, 1),
               hbm_frac_touched=round(by / us_wall / 1e3 / PEAK_HBM_GBPS, 4))
    if dense_us is not None:
        rec["speedup_vs_dense"] = round(dense_us / us_wall, 3)
    return rec, sp, n


def full_form(shape: Shape, r, seed):
    """Device option arrays of the full form (R-S+, SiLU on W_up, G, RMSNorm) for rank r."""
    import torch
    from paper_2609_31975_amd import workloads as wl
    fi = wl.make_form(seed, shape.d, shape.d_ff, r)
    dev = lambda a: torch.from_numpy(a).to("cuda")  # noqa: E731
    return dict(act=1, silu_up=True, g_idx=dev(fi.g_idx), g_sign=dev(fi.g_sign), rms_norm=True,
                rms_gain=dev(fi.rms_gain), rms_eps=1e-6)


def dense_time(shape, r, T, K, W, exact=False, form=None):
    de = Runner(shape, r, T, 1.2816, dense=True, form=form)
    if not exact:
        K = steps_for(de, K)
        W = min(W, K)
    us, _ = time_graph(de, K, W)
    by = algorithmic_bytes(shape.d, shape.d_ff, r, T, shape.d_ff, True, shape.wdt)
    return us, dict(path="lopa_dense" if r else "dense", r=r, T=T, d=shape.d, d_ff=shape.d_ff,
                    us_per_call=round(us, 3), bytes_per_call=int(by),
                    hbm_gbps_touched=round(by / us / 1e3, 1), hbm_frac_touched=round(by / us / 1e3 / PEAK_HBM_GBPS, 4))


def sets_for(per_call_bytes, minimum):
    """Enough weight sets that one rotation touches > 2x the Infinity Cache."""
    need = math.ceil(2 * MALL_BYTES / max(per_call_bytes, 1))
    return max(minimum, need)


# ---------------------------------------------------------------- CPU baseline
def host_cpu():
    """The host CPU's model name and core counts (what the CPU baseline ran on)."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return dict(cpu_model=model, host_cores_visible=len(os.sched_getaffinity(0)), nproc=os.cpu_count())


def cpu_baseline(inp, seed, pool, r, t, seconds, name):
    """The oracle as it stands, on one host core: the sparse method on the headline
    workload for a bounded number of calls (the value; mean and median per call), and the
    dense FFN on three of the same calls (median)."""
    from oracle import ffn_oracle
    from paper_2609_31975_amd import workloads as wl
    xs = wl.make_tokens(seed, pool, inp.d)
    kw = dict(w_gate=inp.w_gate) if r == 0 else dict(lopa_a=inp.lopa_a, lopa_b=inp.lopa_b)
    call = dict(w_up=inp.w_up, w_down_t=inp.w_down_t, t=t, wdt=inp.wdt, **kw)
    ffn_oracle.ffn(xs[:1], **call)  # load + warm
    per = []
    t0 = time.perf_counter()
    while True:
        k = len(per) % len(xs)
        c0 = time.perf_counter()
        ffn_oracle.ffn(xs[k:k + 1], **call)
        per.append(time.perf_counter() - c0)
        el = time.perf_counter() - t0
        if (el >= seconds and len(per) >= 3) or len(per) >= 10000:
            break
    dense = []
    for k in range(3):
        c0 = time.perf_counter()
        ffn_oracle.ffn(xs[k:k + 1], skip_inactive=False, **call)
        dense.append(time.perf_counter() - c0)
    n = len(per)
    return dict(value=round(el * 1e6 / n, 1), unit="us/call", cores=1, kind="oracle",
                sample=f"{n} calls of {name} (weight set 0, tokens 0..{min(n, len(xs)) - 1}), fp64 C oracle, "
                       f"single-threaded, {el:.1f} s; dense oracle on tokens 0..2",
                median_us_per_call=round(float(np.median(per)) * 1e6, 1),
                oracle_dense_us_per_call=round(float(np.median(dense)) * 1e6, 1),
                oracle_dense_sample="3 calls (tokens 0..2), median", **host_cpu())


def torch_dense_time(shape: Shape, T, K, W, t=1.2816):
    """The dense gated FFN written with torch bf16 products (hipBLASLt / rocBLAS GEMMs, bf16
    activations): a sanity column for this library's own dense call.  Weight sets and
    tokens rotate as in the other runners; K calls captured in a graph and timed."""
    import torch
    import torch.nn.functional as F
    s = shape
    xb = [xs.to(torch.bfloat16) for xs in s.x]
    y = torch.empty((T, s.d), dtype=torch.bfloat16, device="cuda")
    batches = s.pool // T

    def run(i):
        k = i % s.n_sets
        b = (i // s.n_sets) % batches
        x = xb[k][b * T:(b + 1) * T]
        h = F.linear(x, s.gate[k])
        v = F.linear(x, s.up[k])
        z = torch.relu(h - t) * v
        torch.matmul(z, s.down[k], out=y)   # [T, d_ff] x [d_ff, d], both contiguous

    class _R:
        torch = __import__("torch")

        def __call__(self, i):
            run(i)
    us, _ = time_graph(_R(), K, W)
    return us


def lopa_approx_record(D, H, r, cpu, log, max_iters=3):
    """Time ffn_lopa_approx on a Gaussian H x D gate (std D^-1/2) at rank r; with `cpu`, the
    oracle (numpy fp64 SVD) on the same matrix, one UV step."""
    import torch
    from paper_2609_31975_amd import ffn
    g = torch.Generator(device="cuda").manual_seed(16)
    w = (torch.randn((H, D), generator=g, device="cuda") * D ** -0.5).contiguous()
    ffn.ffn_lopa_approx(w, r, 1)  # load rocBLAS / rocSOLVER kernels
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    _, _, _, _, it, obj = ffn.ffn_lopa_approx(w, r, max_iters)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    # fp64 work of one UV step: Gram matrix (SYRK, D^2 H), U and the residual (2 x 2 H D r)
    flops = D * D * H + 4.0 * H * D * r
    rec = dict(workload=f"lopa_approx_{H}x{D}_r{r}", path="lopa_approx", H=H, D=D, r=r, uv_steps=it,
               objective=obj, seconds=round(dt, 4), seconds_per_uv_step=round(dt / max(it, 1), 4),
               gemm_tflops_per_step=round(flops / 1e12, 3),
               note="fp64: rocBLAS SYRK/GEMM, rocSOLVER dsyevd (the eigensolver dominates), M step kernel")
    log(f"[bench] lopa approx {H}x{D} r={r}: {dt:.3f} s, {it} UV steps")
    if cpu:
        from oracle import lopa_approx as la
        W = w.cpu().double().numpy()
        t0 = time.perf_counter()
        la.lopa_approx(W, r, max_iters=1)
        rec["cpu_oracle_seconds_one_uv_step"] = round(time.perf_counter() - t0, 3)
        rec["cpu_oracle_cores"] = len(os.sched_getaffinity(0))
        log(f"[bench] lopa approx oracle: {rec['cpu_oracle_seconds_one_uv_step']} s")
    del w
    torch.cuda.empty_cache()
    return rec


def parity_sample(shape: Shape, r, T, t, form=None, form_seed=None):
    """Step 0 of the timed workload (weight set 0, its first T tokens, the same call and
    launch configuration): relative error of every token's output against the oracle,
    and the active union against the union of the oracle's per-token active sets (a
    neuron within 1e-3 of t for some token may go either way)."""
    import torch
    from oracle import ffn_oracle
    from paper_2609_31975_amd import ffn
    from paper_2609_31975_amd import workloads as wl
    inp = shape.host0[r]
    run = Runner(shape, r, T, t, dense=False, form=form)
    run(0)
    torch.cuda.synchronize()
    y = run.y.cpu().numpy().astype(np.float64)
    x = run.args(0)[1].cpu().numpy()
    kw = dict(w_gate=inp.w_gate) if r == 0 else dict(lopa_a=inp.lopa_a, lopa_b=inp.lopa_b)
    if inp.scales is not None:
        kw["scales"] = inp.scales
    if form is not None:
        fi = wl.make_form(form_seed, shape.d, shape.d_ff, r)
        kw.update(act=form["act"], silu_up=form["silu_up"], g_idx=fi.g_idx, g_sign=fi.g_sign,
                  rms_norm=form["rms_norm"], rms_gain=fi.rms_gain, rms_eps=form["rms_eps"])
    res = ffn_oracle.ffn(x, w_up=inp.w_up, w_down_t=inp.w_down_t, t=t, wdt=inp.wdt, **kw)
    idx, _ = ffn.ffn_active_set(run.ws, T, shape.d, shape.d_ff, r, with_act=False)
    ref = np.flatnonzero(res.active.any(0))
    band = (np.abs(res.h - np.float32(t)) < 1e-3).any(0)
    mism = np.setxor1d(idx, ref)
    err = [float(np.linalg.norm(y[k] - res.y[k]) / max(np.linalg.norm(res.y[k]), 1e-300)) for k in range(T)]
    return dict(tokens=T, rel_err=max(err),
                active_set_mismatches_outside_band=int((~band[mism]).sum()) if len(mism) else 0)


def copy_calibration(K):
    """A plain elementwise kernel of known size (reads and writes 256 MiB), for scaling
    the HBM byte counters."""
    import torch
    n = 256 << 20
    src = torch.ones(n // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(K):
        torch.neg(src, out=dst)
    torch.cuda.synchronize()
    return dict(kernel="neg", bytes_read=n, bytes_written=n, launches=K)


# sources the T = 1 kernels are built from (the batched kernels live in ffn_batched.hip)
T1_SOURCES = ("ffn_device.h", "ffn_internal.h", "ffn_kernels.hip")


def kernel_source_digest():
    """sha256 over the sources of the dominant kernel (in a fixed order): a counter
    profile holds for the kernel it was taken on only."""
    import hashlib
    csrc = os.path.join(ROOT, "paper_2609_31975_amd", "csrc")
    h = hashlib.sha256()
    for f in T1_SOURCES:
        h.update(f.encode() + b"\0" + open(os.path.join(csrc, f), "rb").read())
    return h.hexdigest()


def recorded_traffic(workload):
    """HBM bytes per launch of the dominant kernel from the committed counter profile
    (profiles/<kernel>_<workload>_pmc.json), or None if the kernels changed since."""
    path = os.path.join(ROOT, "profiles", f"k_gate_up_t1_{workload}_pmc.json")
    if not os.path.exists(path):
        return None, None
    rec = json.load(open(path))
    if rec.get("kernel_source_sha256") != kernel_source_digest():
        return None, path
    return int(rec["traffic_bytes"]), path


# ---------------------------------------------------------------- main
def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the sparse FFN hot path here is a single-GPU kernel "
              "sequence and the library runs no collectives; use --gpus 1", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2609_31975_amd import ffn
    from paper_2609_31975_amd import workloads as wl
    ffn.lib()  # fail loudly if the HIP library is missing
    assert torch.cuda.is_available(), "bench.py needs a ROCm GPU"
    torch.cuda.set_device(0)
    K, W = args.steps, args.warmup
    head = wl.workload(args.workload)

    def log(*a):
        print(*a, file=sys.stderr, flush=True)

    shapes = {}

    def get_shape(d, d_ff, ranks, n_sets, seed, pool=64, wdt=wl.BF16):
        key = (d, d_ff, wdt)
        if key not in shapes:
            shapes.clear()
            torch.cuda.empty_cache()
            log(f"[bench] generating {n_sets} weight sets d={d} d_ff={d_ff} ranks={ranks} format={wdt}")
            shapes[key] = Shape(d, d_ff, ranks, n_sets, seed, pool, wdt=wdt)
        return shapes[key]

    def family_sets(d, d_ff, minimum):
        """Weight sets for one shape: enough that the LoPA rotation (the smallest per-call
        footprint of the family) exceeds twice the Infinity Cache."""
        rank = 512 if d == 4096 else 1024
        return max(sets_for(algorithmic_bytes(d, d_ff, 0, 1, 0.1 * d_ff, False), minimum),
                   sets_for(algorithmic_bytes(d, d_ff, rank, 1, 0.1 * d_ff, False), minimum))

    # ---- headline
    r0, T0 = head.r, head.T
    rank = 512 if head.d == 4096 else 1024
    ranks = sorted({0, rank, r0}) if not args.no_sweep else sorted({0, r0})
    sh = get_shape(head.d, head.d_ff, ranks, family_sets(head.d, head.d_ff, head.n_sets), head.seed, pool=256,
                   wdt=head.wdt)
    log(f"[bench] headline {head.name}: {sh.n_sets} sets, K={K}, W={W}")
    hform = full_form(sh, r0, head.seed) if head.form == "full" else None
    dense_us, dense_rec = dense_time(sh, 0, T0, K, W, exact=True)
    rec, run, nlist = measure(sh, r0, T0, head.t, K, W, dense_us=dense_us, name=head.name, exact=True, form=hform,
                              rho=head.rho)
    gate_mean, gate_med = time_gate_kernel(run, K)
    flushed = time_flushed(run)
    gbytes = np.mean([gate_kernel_bytes(head.d, head.d_ff, r0, T0, k, False, head.wdt) for k in nlist])
    par = parity_sample(sh, r0, T0, head.t, form=hform, form_seed=head.seed)
    traffic, traffic_src = recorded_traffic(head.name)
    log(f"[bench] headline {rec['us_per_call']} us/call, dense {dense_us:.2f}, gate kernel {gate_mean:.2f} us, "
        f"parity {par}")
    kernel = "k_gate_up_t1 (gate GEMV + threshold + compaction + W_up rows)" if T0 == 1 else \
        "k_gate_up_mfma (gate + union + W_up rows, matrix cores)"
    out = {
        "metric": METRIC,
        "value": rec["us_per_call"],
        "unit": "us/call",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": round(rec["us_per_call"] / 1e3, 6),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        # the paper's own FFN-only GPU speedups (Section 5.3), context only: its 5.8B-parameter
        # model on a GPU the paper does not name, not this workload or machine
        "paper_context": {"speedup_vs_dense": {"standard_s90": 2.06, "lopa_s90": 3.31, "lopa_s95": 3.90},
                          "model": "5.8B parameters (FFN only)", "gpu": "not stated in the paper"},
        "dtype": "f32",
        "weight_dtype": {0: "f32", 1: "bf16", 2: "int8", 3: "int4"}[head.wdt],
        "data": "synthetic: seeded Gaussian weights (N(0,1/d), W_down N(0,1/d_ff)), iid N(0,1) tokens",
        "config": {"workload": head.name, "d": head.d, "d_ff": head.d_ff, "T": T0, "gating": "lopa" if r0 else
                   "standard", "r": r0, "t": head.t, "weight_sets": sh.n_sets, "timing": "HIP graph of K calls"},
        "speedup_vs_dense": rec.get("speedup_vs_dense"),
        "dense_us_per_call": round(dense_us, 3),
        "n_active": rec["n_union"],
        "bytes_per_call": rec["bytes_per_call"],
        "hbm_gbps_touched": rec["hbm_gbps_touched"],
        "hbm_frac_touched": rec["hbm_frac_touched"],
        "roofline": {"bound": "hbm", "kernel": kernel, "scope": "dominant kernel only",
                     "achieved": round(gbytes / gate_mean / 1e3, 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                     "frac": round(gbytes / gate_mean / 1e3 / PEAK_HBM_GBPS, 4), "traffic": traffic,
                     "bytes_per_launch": int(gbytes), "avg_duration_us": round(gate_mean, 3),
                     "median_duration_us": round(gate_med, 3),
                     "traffic_source": (os.path.relpath(traffic_src, ROOT) if traffic_src else None),
                     "call_level_frac": rec["hbm_frac_touched"]},
        "parity_sample": par,
        "us_per_call_events": rec["us_per_call_events"],
        # eager calls, each after a 1 GiB write (Infinity Cache and L2 cold), median
        "us_per_call_mall_flushed": round(flushed, 3),
    }

    # ---- sweep
    sweep = [dict(rec, path="sparse"), dict(dense_rec, workload=head.name)]
    host_head = sh.host0[r0]
    del run

    def sweep_family(shp, works, k, w_, dense_t1):
        """Every workload of one shape, each with its dense baselines (the library's dense
        call, the LoPA gate with every neuron, and the dense FFN in torch bf16 products)."""
        dense = {1: dense_t1} if dense_t1 is not None else {}
        tdense = {}
        for w in works:
            form = full_form(shp, w.r, w.seed) if w.form == "full" else None
            rw, rrun, _ = measure(shp, w.r, w.T, w.t, k, w_, name=w.name, form=form, rho=w.rho)
            if w.T == 1:
                rw["us_per_call_mall_flushed"] = round(time_flushed(rrun), 3)
            del rrun
            if w.rho:
                rw["token_correlation"] = w.rho
                base = [q for q in sweep if q.get("workload") == f"8b_lopa512_s90_T{w.T}"]
                if base:
                    rw["iid_us_per_call"] = base[0]["us_per_call"]
                    rw["iid_union"] = base[0]["n_union"]
            if form is not None:
                rw["form"] = "full: R-S+ activation, SiLU on W_up, G term, RMSNorm between A and B"
                base = [q for q in sweep if q.get("workload") == f"8b_lopa512_s90_T{w.T}"]
                if base:
                    rw["default_form_us_per_call"] = base[0]["us_per_call"]
            if w.T not in dense:
                dense[w.T] = dense_time(shp, 0, w.T, k, w_)[0]
            if w.T not in tdense and shp.wdt == wl.BF16:
                tdense[w.T] = torch_dense_time(shp, w.T, k, w_)
            du = dense[w.T]
            rw["dense_us_per_call"] = round(du, 3)
            rw["speedup_vs_dense"] = round(du / rw["us_per_call"], 3)
            if w.T in tdense:
                rw["torch_bf16_dense_us_per_call"] = round(tdense[w.T], 3)
            if w.r:
                ldu, _ = dense_time(shp, w.r, w.T, k, w_, form=form)
                rw["lopa_dense_us_per_call"] = round(ldu, 3)
                rw["speedup_vs_lopa_dense"] = round(ldu / rw["us_per_call"], 3)
            rw["path"] = "sparse"
            sweep.append(rw)
            log(f"[bench] {w.name}: {rw['us_per_call']} us, x{rw['speedup_vs_dense']} vs dense")
        return tdense

    if not args.no_sweep:
        bf16 = [w for w in wl.workloads() if w.wdt == wl.BF16]
        fam = [w for w in bf16 if w.d == head.d and w.name != head.name]
        kf = K if head.d == 4096 else max(K // 4, 20)
        wf = W if head.d == 4096 else max(W // 4, 5)
        td = sweep_family(sh, fam, kf, wf, dense_us if T0 == 1 else None)
        if T0 in td:
            out["torch_bf16_dense_us_per_call"] = round(td[T0], 3)
        elif head.wdt == wl.BF16:
            out["torch_bf16_dense_us_per_call"] = round(torch_dense_time(sh, T0, kf, wf), 3)
        shapes.clear()
        torch.cuda.empty_cache()
        # the other shape family (8B-shaped after a 70B headline, or the reverse)
        od, odff = (4096, 14336) if head.d != 4096 else (8192, 28672)
        other = [w for w in bf16 if w.d == od]
        if other:
            k2, w2 = (K, W) if od == 4096 else (max(K // 4, 20), max(W // 4, 5))
            r2 = 512 if od == 4096 else 1024
            sh2 = get_shape(od, odff, [0, r2], family_sets(od, odff, other[0].n_sets), other[0].seed, pool=256)
            sweep_family(sh2, other, k2, w2, None)
            shapes.clear()
            torch.cuda.empty_cache()
        # quantized weights (8B shape): sparse and dense in the same format; single-token
        # calls also against the bf16 dense call and an fp32 dense call (the paper's
        # full-precision baseline)
        bf16_dense_8b = next((q["dense_us_per_call"] for q in sweep if q.get("workload") == "8b_std_s90"), None)
        qw = [w for w in wl.workloads() if w.wdt in wl.QMAX]
        if qw:
            f32 = Shape(4096, 14336, [0], sets_for(algorithmic_bytes(4096, 14336, 0, 1, 14336, True, wl.F32), 2),
                        qw[0].seed, 64, wdt=wl.F32)
            f32_us, _ = dense_time(f32, 0, 1, K, W)
            del f32
            torch.cuda.empty_cache()
            log(f"[bench] fp32 dense {f32_us:.2f} us")
            for wdt in sorted({w.wdt for w in qw}):
                ws_ = [w for w in qw if w.wdt == wdt]
                per = algorithmic_bytes(4096, 14336, 0, 1, 0.1 * 14336, False, wdt)
                shq = Shape(4096, 14336, sorted({0} | {w.r for w in ws_}), sets_for(per, 4), ws_[0].seed, 64, wdt=wdt)
                qdense = {}
                for w in ws_:
                    rw = measure(shq, w.r, w.T, w.t, K, W, name=w.name)[0]
                    if (w.r, w.T) not in qdense:
                        qdense[(w.r, w.T)] = dense_time(shq, w.r, w.T, K, W)[0]
                    qd = qdense[(w.r, w.T)]
                    rw.update(weights={wl.I8: "int8", wl.I4: "int4"}[wdt], path="sparse",
                              dense_same_format_us_per_call=round(qd, 3),
                              speedup_vs_dense_same_format=round(qd / rw["us_per_call"], 3))
                    if w.T == 1:  # the bf16 and fp32 dense calls are single-token ones
                        if bf16_dense_8b:
                            rw.update(dense_us_per_call=bf16_dense_8b,
                                      speedup_vs_dense=round(bf16_dense_8b / rw["us_per_call"], 3))
                        rw.update(fp32_dense_us_per_call=round(f32_us, 3),
                                  speedup_vs_fp32_dense=round(f32_us / rw["us_per_call"], 3))
                        log(f"[bench] {w.name}: {rw['us_per_call']} us, x{rw.get('speedup_vs_dense')} vs bf16 dense, "
                            f"x{rw['speedup_vs_fp32_dense']} vs fp32 dense")
                    else:
                        log(f"[bench] {w.name}: {rw['us_per_call']} us, x{rw['speedup_vs_dense_same_format']} vs "
                            f"dense in the same format")
                    sweep.append(rw)
                del shq
                torch.cuda.empty_cache()
        # the tiny fp32 workload: L2-resident and launch-bound, so its byte rate means nothing
        for w in [w for w in wl.workloads() if w.name.startswith("tiny")]:
            sht = Shape(w.d, w.d_ff, [0], 1, w.seed, 64, wdt=w.wdt)
            tdu, _ = dense_time(sht, 0, 1, K, W)
            rw = measure(sht, 0, 1, w.t, K, W, dense_us=tdu, name=w.name)[0]
            rw.update(path="sparse", dense_us_per_call=round(tdu, 3),
                      note="L2-resident (3 MB of weights, one set): launch-bound, the byte rate is not an HBM figure")
            sweep.append(rw)
            log(f"[bench] {w.name}: {rw['us_per_call']} us, x{rw['speedup_vs_dense']} vs dense")
            del sht
        # LoPA approximation of the 8B gate (Section 3.3): one conversion, timed end to end
        sweep.append(lopa_approx_record(4096, 14336, 512, cpu=not args.no_cpu, log=log))
    out["sweep"] = sweep

    # ---- CPU baseline (oracle, host cores) on the headline workload
    if not args.no_cpu:
        out["cpu_baseline"] = cpu_baseline(host_head, head.seed, sh.pool, r0, head.t, args.cpu_seconds, head.name)
        log(f"[bench] cpu baseline {out['cpu_baseline']['value']} us/call (dense oracle "
            f"{out['cpu_baseline']['oracle_dense_us_per_call']} us/call)")
    else:
        out["cpu_baseline"] = None
    if args.copy_calibration:
        out["copy_calibration"] = copy_calibration(5)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
