"""Benchmark of the SSBA forward path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload grid64]
                    [--no-cpu] [--sweep] [--copy-calibration] [--layers] [--haar]
                    [--backward]

One step = one SSBA layer call on inputs already resident in HBM: the top-k
gate (block pooling, affinity, ranking -> index) and the block-sparse
attention, through ssba_forward_topk (pooling of K, then the attention
kernel, which gates each query block itself and writes the index).  The
same call as ssba_build_index + ssba_forward is timed too
(ms_step_two_calls).  Steps run back to back between two HIP events on the
stream the library launches on, once launched eagerly and once replayed from
a HIP graph captured from the same calls (same kernels, same work; the replay
is checked bit-exact against the eager output); `value` uses the faster.
Index, forward and dense launches, and the two-call form, are also timed
separately, back to back: five rounds that time each form in turn, median
per form.  Before the warm-up steps, a clock-settle phase runs the step back
to back for --settle-ms milliseconds of wall time (default 100): the GPU
clock needs about 10 ms of load to reach its steady state, and without the
phase the first timed milliseconds run 10-15 % slow.  The phase is reported
in the output line (clock_settle_ms, clock_settle_calls); --settle-ms 0
switches it off.
These are warm numbers (Q, K, V and O stay in the 256 MB MALL between
calls); ms_step_cold and ms_fwd_cold are the median of ten single calls each
made after a 1 GiB buffer is written, so the inputs come from HBM.  Prints
ONE JSON line on stdout; --sweep prints extra per-configuration lines on
stderr (sparsity sweep, text tokens, 2K grid).

Flops are counted over computed (kept) query/key pairs only: 4 * D per pair
(2 * D for Q K^T, 2 * D for P V).  Pairs per (batch, head):
T_img * (keep * Bt^2 + T_txt) + T_txt * T.

The roofline object describes the step's dominant kernel: the gated
attention launch of ssba_forward_topk (the attention kernel with the top-k
gate of each query block in its prologue), timed alone through
ssba_forward_gated_ex on the pooled key sums the step's pooling launch left
in the scratch: its flops per launch over its average launch time (HIP
events on the stream it runs on).  roofline_ungated gives the same for the
attention kernel as ssba_forward launches it (index read, no gate), and
ms_pool the pooling launch alone.  ms_step_rope times Algorithm 1 in full,
its rotary step included (ssba_forward_topk_rope_ex: the rotary pre-pass,
which writes the rotated Q and K and pools the rotated keys, then the gated
attention on them), and ms_rope_pool / gbs_rope_pool that pre-pass alone
against its compulsory bytes.  `traffic` is the HBM traffic per launch
measured with rocprofv3 counters (FETCH_SIZE and WRITE_SIZE, scaled by what
the same counters read for a plain copy of known size), reported only while
the kernel's sources still hash to the values the counters were taken on.

--layers prints instead one JSON line for a 24-layer stack through
ssba_forward_layers (synthetic per-layer keep schedule averaging 84.18 %
masked, the offset alternating with layer parity, distinct inputs per layer):
the stack, the same layers as separate calls, a depth-pruned stack, the
head-shared gate and the window gate with its per-parity index cache.

--haar prints instead one JSON line for the multi-level Haar transform pair
(T-DVAE wavelets) on a [1, 128, 512, 512] bf16 feature map, 3 levels: the
forward and inverse launch times and their GB/s against the HBM roofline.

--backward prints instead one JSON line for a training step of the call:
the forward with its log-sum-exp and the backward (dQ, dK, dV with the gate
held fixed), TFLOP/s counting 10 D flops per computed pair in the backward.

--copy-calibration runs only that plain copy (256 MiB, 5 times) for the
counter runs and prints its size.
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import statistics
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0
COPY_BYTES = 256 << 20
REPEATS = 5                 # rounds of the companion timings (median)

# HBM traffic per launch from counter runs, keyed by kernel and workload:
# the sources the kernel was built from (sha256 over their bytes, in order),
# FETCH_SIZE and WRITE_SIZE in KiB per dispatch, and the copy calibration
# factors (bytes known / bytes the counter reads for a plain 256 MiB copy).
# From the counter summary in profiles/k_attn_mfma_grid64.md.
MEASURED_TRAFFIC = {
    ("k_haar_dwt<unsigned short, 3>", "haar512"): {"sha": "02be9c317bd1aa8b", "fetch_kib": 131115.0,
                                                  "write_kib": 344064.0, "fetch_factor": 1.9998,
                                                  "write_factor": 1.0},
    ("k_attn_mfma<64, 3, false, true>", "grid64"): {"sha": "5c3b7efa87c23894", "fetch_kib": 12668.0,
                                                    "write_kib": 8456.0, "fetch_factor": 1.99984,
                                                    "write_factor": 1.0},
    ("k_attn_mfma<64, 3, false, false>", "grid64"): {"sha": "5c3b7efa87c23894", "fetch_kib": 12554.8,
                                                     "write_kib": 8192.0, "fetch_factor": 1.99984,
                                                     "write_factor": 1.0},
}

def kernel_sources(kernel: str):
    base = os.path.join(ROOT, "paper_2605_15684_amd", "csrc")
    stem = kernel.split("<")[0]
    if stem in ("k_haar_dwt", "k_haar_iwt"):
        return [os.path.join(base, "ssba_haar.hip"), os.path.join(ROOT, "include", "ssba_haar.h")]
    own = {"k_attn_mfma": "ssba_attn_mfma.hip", "k_attn_bf16": "ssba_attn_bf16.hip",
           "k_attn_f32": "ssba_attn_f32.hip"}[stem]
    return [os.path.join(base, own), os.path.join(base, "ssba_common.h"),
            os.path.join(ROOT, "include", "ssba.h")]


def sources_sha(kernel: str) -> str:
    import hashlib
    h = hashlib.sha256()
    for f in kernel_sources(kernel):
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch, or None if not measured on these sources."""
    m = MEASURED_TRAFFIC.get((kernel, workload))
    if not m or m["sha"] != sources_sha(kernel):
        return None
    return m["fetch_kib"] * 1024 * m["fetch_factor"] + m["write_kib"] * 1024 * m["write_factor"]


def rope_bytes(w) -> int:
    """Compulsory bytes of the rotary pre-pass: Q and K read, rotated Q and K
    written, the pooled key sums written (bf16 tensors, fp64 sums)."""
    return 4 * w.batch * w.heads * w.seq_len * w.head_dim * 2 + w.batch * w.heads * w.n_tiles * w.head_dim * 8


def pairs_per_bh(w, keep=None) -> int:
    keep = w.keep if keep is None else keep
    if w.gate == "window":
        keep = w.window[0] * w.window[1]
    elif w.gate == "dense":
        keep = w.n_tiles
    return w.t_img * (keep * w.tile * w.tile + w.n_text) + w.n_text * w.seq_len


def flops(w, dense=False) -> float:
    pairs = w.seq_len * w.seq_len if dense else pairs_per_bh(w)
    return 4.0 * w.head_dim * pairs * w.batch * w.heads


def describe(w) -> str:
    s = f"B{w.batch} H{w.heads} {w.grid_h}x{w.grid_w} tokens D{w.head_dim} {w.tile}x{w.tile} blocks"
    if w.gate == "topk":
        s += f" top-k keep {w.keep}/{w.n_tiles} ({100 * (1 - w.keep / w.n_tiles):.3f}% masked)"
    elif w.gate == "window":
        s += f" window {w.window[0]}x{w.window[1]} blocks"
    else:
        s += " dense gate"
    if w.n_text:
        s += f" + {w.n_text} dense text tokens"
    return s + f" shift {w.shift} bf16 seed {w.seed}"


class Runner:
    """Preallocated buffers and the timed calls of one workload."""

    def __init__(self, w):
        import torch
        from paper_2605_15684_amd import ssba
        from paper_2605_15684_amd.inputs import make_qkv
        self.torch, self.ssba, self.w = torch, ssba, w
        self.q, self.k, self.v = make_qkv(w, device="cuda")
        self.desc = ssba.desc_for(self.q, grid=(w.grid_h, w.grid_w), tile=w.tile, shift=w.shift,
                                  n_text=w.n_text, gate=w.gate, keep=w.keep, window=w.window)
        self.index, self.scratch = ssba.alloc_workspace(self.desc, self.q.device)
        self.out = torch.empty_like(self.q)
        self.out_dense = torch.empty_like(self.q)

    def fused(self) -> bool:
        """True when the step is the fused form (pooling launch + gated attention)."""
        from paper_2605_15684_amd import _lib
        return self.w.gate == "topk" and _lib.forward_kernel(self.desc, mode=2) != \
            _lib.forward_kernel(self.desc, mode=0)

    def step(self):
        """One layer call: ssba_forward_topk (gate fused into attention) for
        the top-k gate; the static gates go through the two-call form."""
        if self.w.gate != "topk":
            return self.step_two_calls()
        self.ssba.forward_topk(self.q, self.k, self.v, self.desc, self.index, self.scratch, self.out)

    def step_two_calls(self):
        """The same layer call as ssba_build_index then ssba_forward."""
        self.ssba.build_index(self.q, self.k, self.desc, self.index, self.scratch)
        self.ssba.forward(self.q, self.k, self.v, self.index, self.desc, self.out)

    def _span(self, fn, steps: int) -> float:
        """Milliseconds per call of `fn`: HIP events on the current stream (the
        one the library launches on) around `steps` back-to-back calls."""
        torch = self.torch
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(steps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps

    def run_index(self):
        self.ssba.build_index(self.q, self.k, self.desc, self.index, self.scratch)

    def run_fwd(self):
        self.ssba.forward(self.q, self.k, self.v, self.index, self.desc, self.out)

    def run_dense(self):
        self.ssba.forward_dense(self.q, self.k, self.v, self.desc, self.out_dense)

    def run_pool(self):
        """The step's pooling launch alone (ssba_pool_keys_ex)."""
        self.ssba.pool_keys(self.k, self.desc, self.scratch)

    def run_gated(self):
        """The step's gated attention launch alone (ssba_forward_gated_ex), on
        the pooled key sums the last step or run_pool left in the scratch."""
        self.ssba.forward_gated(self.q, self.k, self.v, self.desc, self.index, self.scratch, self.out)

    def run_rope_step(self):
        """Algorithm 1 in full, rotary step included (ssba_forward_topk_rope_ex)."""
        if not hasattr(self, "q_rope"):
            self.q_rope, self.k_rope = self.torch.empty_like(self.q), self.torch.empty_like(self.k)
        self.ssba.forward_topk_rope(self.q, self.k, self.v, self.desc, q_rope=self.q_rope, k_rope=self.k_rope,
                                    index=self.index, scratch=self.scratch, out=self.out)

    def run_rope_pool(self):
        """Its rotary pre-pass alone (ssba_rope_pool_keys_ex)."""
        if not hasattr(self, "q_rope"):
            self.q_rope, self.k_rope = self.torch.empty_like(self.q), self.torch.empty_like(self.k)
        self.ssba.rope_pool_keys(self.q, self.k, self.desc, self.scratch, q_rope=self.q_rope, k_rope=self.k_rope)

    def timed_steps(self, steps: int):
        """Whole steps (index + forward) back to back: wall ms and event ms per step."""
        torch = self.torch
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        ms = self._span(self.step, steps)
        wall = (time.perf_counter() - t0) * 1e3 / steps
        return wall, ms

    def cold_ms(self, fn, reps: int = 10) -> float:
        """Median ms of one call of `fn` after a 1 GiB buffer is written, which
        evicts Q, K, V and O from the 256 MB last-level cache (MALL)."""
        torch = self.torch
        if not hasattr(self, "_evict"):
            self._evict = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
        times = []
        for r in range(reps):
            self._evict.fill_(float(r))
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            times.append(e0.elapsed_time(e1))
        times.sort()
        return times[len(times) // 2]

    def graph_step_ms(self, steps: int):
        """The same step captured once in a HIP graph and replayed."""
        torch = self.torch
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            for _ in range(3):
                self.step()
        torch.cuda.current_stream().wait_stream(side)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            self.step()
        g.replay()
        ms = self._span(g.replay, steps)
        return ms, g


def cpu_model() -> str:
    """Host CPU model name from /proc/cpuinfo (platform's processor string
    otherwise)."""
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or platform.machine()


def cpu_baseline(runner, budget_s: float = 12.0) -> dict:
    """The fp64 oracle on the same inputs: the gate for every (batch, head),
    then attention head by head until the time budget is spent."""
    import torch
    from oracle import ssba_oracle as O
    w = runner.w
    q = runner.q.double().cpu().numpy()
    k = runner.k.double().cpu().numpy()
    v = runner.v.double().cpu().numpy()
    kw = dict(grid_h=w.grid_h, grid_w=w.grid_w, tile=w.tile, shift=w.shift, n_text=w.n_text)
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = 1
    t0 = time.perf_counter()
    idx = O.build_index(q, k, gate=w.gate, keep=w.keep, window=w.window, **kw)
    t_index = time.perf_counter() - t0
    n_bh = w.batch * w.heads
    done, t_attn = 0, 0.0
    for bh in range(n_bh):
        b, h = divmod(bh, w.heads)
        t1 = time.perf_counter()
        O.attention(q, k, v, idx, heads=[(b, h)], **kw)
        t_attn += time.perf_counter() - t1
        done += 1
        if t_index + t_attn > budget_s:
            break
    per_bh = flops(w) / n_bh
    sec = t_index * done / n_bh + t_attn
    return {"value": per_bh * done / sec / 1e12, "unit": "TFLOP/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"fp64 oracle: gate for all {n_bh} (batch, head) pairs "
                      f"({t_index:.2f} s, pro-rated), attention for {done} of {n_bh} pairs "
                      f"({t_attn:.2f} s); host {cpu_model()}, os.cpu_count()={os.cpu_count()}",
            "cpu_model": cpu_model(),
            "seconds": round(t_index + t_attn, 3)}


def settle_clock(fn, ms: float) -> int:
    """Run `fn` back to back for `ms` milliseconds of wall time (synchronizing
    every 50 calls); returns the number of calls."""
    import torch
    calls = 0
    t0 = time.perf_counter()
    while (time.perf_counter() - t0) * 1e3 < ms:
        for _ in range(50):
            fn()
        calls += 50
        torch.cuda.synchronize()
    return calls


def measure(w, steps: int, warmup: int, dense_steps: int, graph: bool = True, settle_ms: float = 0.0):
    r = Runner(w)
    settle_calls = settle_clock(r.step, settle_ms) if settle_ms > 0 else 0
    for _ in range(warmup):
        r.step()
    wall_ms, step_ms = r.timed_steps(steps)
    # The companion timings: five rounds, each timing every call form once in
    # turn, and the median per form, so that no form is favoured by its place
    # in the sequence (the clock settles over the first milliseconds of load).
    for _ in range(3):
        r.run_dense()
    fused = r.fused()
    spans = {"two": [], "idx": [], "fwd": [], "dense": [], "gated": [], "pool": [], "rope": [], "rope_pool": []}
    for _ in range(REPEATS):
        spans["two"].append(r._span(r.step_two_calls, steps))
        spans["idx"].append(r._span(r.run_index, steps))
        spans["fwd"].append(r._span(r.run_fwd, steps))
        spans["dense"].append(r._span(r.run_dense, dense_steps))
        if fused:
            spans["pool"].append(r._span(r.run_pool, steps))
            spans["gated"].append(r._span(r.run_gated, steps))
            spans["rope"].append(r._span(r.run_rope_step, steps))
            spans["rope_pool"].append(r._span(r.run_rope_pool, steps))
    two_ms, idx_ms, fwd_ms, dense_ms = (statistics.median(spans[key])
                                        for key in ("two", "idx", "fwd", "dense"))
    gated_ms = statistics.median(spans["gated"]) if fused else None
    pool_ms = statistics.median(spans["pool"]) if fused else None
    rope_ms = statistics.median(spans["rope"]) if fused else None
    rope_pool_ms = statistics.median(spans["rope_pool"]) if fused else None
    cold_step_ms = r.cold_ms(r.step)
    cold_fwd_ms = r.cold_ms(r.run_fwd)
    graph_ms = None
    if graph:
        graph_ms, g = r.graph_step_ms(steps)
        # the graph's outputs must equal the eager ones bit for bit
        ref = r.out.clone()
        g.replay()
        r.torch.cuda.synchronize()
        assert r.torch.equal(ref, r.out), "graph replay differs from eager step"
        del g
    best_ms = min(step_ms, graph_ms) if graph_ms is not None else step_ms
    f = flops(w)
    return r, {
        "ms_step_wall": wall_ms, "ms_step_eager": step_ms, "ms_step_graph": graph_ms,
        "ms_step": best_ms, "ms_step_two_calls": two_ms, "ms_index": idx_ms, "ms_fwd": fwd_ms,
        "ms_dense": dense_ms, "ms_gated": gated_ms, "ms_pool": pool_ms, "ms_step_rope": rope_ms,
        "ms_rope_pool": rope_pool_ms, "ms_step_cold": cold_step_ms,
        "ms_fwd_cold": cold_fwd_ms, "gflop": f / 1e9, "gflop_dense": flops(w, dense=True) / 1e9,
        "tflops_fwd": f / (fwd_ms * 1e-3) / 1e12,
        "tflops_step": f / (best_ms * 1e-3) / 1e12,
        "tflops_dense": flops(w, dense=True) / (dense_ms * 1e-3) / 1e12,
        "speedup_kernel": dense_ms / fwd_ms, "speedup_step": dense_ms / best_ms,
        "settle_calls": settle_calls,
    }


def measured_mfma_tflops(blocks: int = 1024, iters: int = 2000, reps: int = 3) -> float:
    """bf16 MFMA throughput the chip sustains in this process: the library's
    probe (back-to-back v_mfma_f32_32x32x16_bf16, four waves per SIMD), best
    of `reps` launches timed with HIP events on the stream it runs on."""
    import torch
    from paper_2605_15684_amd import _lib
    sink = torch.empty(blocks * 256, dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    _lib.check(_lib.probe_mfma(blocks, 10, sink.data_ptr(), stream), "ssba_probe_mfma")
    best = float("inf")
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        _lib.check(_lib.probe_mfma(blocks, iters, sink.data_ptr(), stream), "ssba_probe_mfma")
        e1.record()
        torch.cuda.synchronize()
        best = min(best, e0.elapsed_time(e1))
    return blocks * 4 * iters * 8 * 32768 / (best * 1e-3) / 1e12


def measure_layers(w, steps: int, warmup: int, settle_ms: float = 0.0) -> dict:
    """A 24-layer stack through ssba_forward_layers: the synthetic per-layer
    keep schedule, the offset alternating by layer parity, every layer with
    its own seeded Q, K, V (so the stack's 768 MB do not fit the MALL).  The
    stack and the same layers as separate calls are timed in alternation,
    REPEATS rounds, median of each, after the clock-settle phase."""
    import torch
    from paper_2605_15684_amd import ssba
    from paper_2605_15684_amd.inputs import LAYER_KEEP_SCHEDULE_24, LAYER_SKIP_24, make_qkv
    keeps = LAYER_KEEP_SCHEDULE_24
    layers = []
    for l, kp in enumerate(keeps):
        q, k, v = make_qkv(w.with_(seed=w.seed + 100 + l), device="cuda")
        layers.append(dict(q=q, k=k, v=v, out=torch.empty_like(q), keep=kp))
    desc = ssba.desc_for(layers[0]["q"], grid=(w.grid_h, w.grid_w), tile=w.tile, shift=w.shift,
                         n_text=w.n_text, gate="topk", keep=keeps[0])

    def span(fn, n):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(n):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    index, scratch = ssba.forward_layers(layers, desc)
    stack = lambda: ssba.forward_layers(layers, desc, index, scratch)
    settle_calls = settle_clock(stack, settle_ms) if settle_ms > 0 else 0

    # The same layers as 24 separate fused calls from Python.
    per = []
    for l, L in enumerate(layers):
        dl = ssba.desc_for(L["q"], grid=(w.grid_h, w.grid_w), tile=w.tile,
                           shift=ssba.layer_shift(l, w.tile), n_text=w.n_text, gate="topk", keep=keeps[l])
        il, sl = ssba.alloc_workspace(dl, L["q"].device)
        per.append((L, dl, il, sl))

    def separate():
        for L, dl, il, sl in per:
            ssba.forward_topk(L["q"], L["k"], L["v"], dl, il, sl, L["out"])
    rounds = {"stack": [], "separate": []}
    for _ in range(REPEATS):
        rounds["stack"].append(span(stack, steps))
        rounds["separate"].append(span(separate, steps))
    ms_stack = statistics.median(rounds["stack"])
    ms_separate = statistics.median(rounds["separate"])

    # Depth-pruned stack: the skip mask of the bench (6 of 24 layers skipped).
    pruned = [dict(L, skip=sk) for L, sk in zip(layers, LAYER_SKIP_24)]
    ms_pruned = span(lambda: ssba.forward_layers(pruned, desc, index, scratch), steps)

    # Head-shared gate on the same stack.
    d_sh = ssba.desc_for(layers[0]["q"], grid=(w.grid_h, w.grid_w), tile=w.tile, shift=w.shift,
                         n_text=w.n_text, gate="topk_shared", keep=keeps[0])
    i_sh, s_sh = ssba.forward_layers(layers, d_sh)
    ms_shared = span(lambda: ssba.forward_layers(layers, d_sh, i_sh, s_sh), steps)

    # Window gate (4x4 blocks, 75 % masked): the index is built once per parity.
    d_win = ssba.desc_for(layers[0]["q"], grid=(w.grid_h, w.grid_w), tile=w.tile, shift=w.shift,
                          n_text=w.n_text, gate="window", window=(4, 4))
    i_w, s_w = ssba.forward_layers(layers, d_win)
    ms_window = span(lambda: ssba.forward_layers(layers, d_win, i_w, s_w), steps)

    gf = sum(flops(w.with_(keep=kp)) for kp in keeps)
    gf_pruned = sum(flops(w.with_(keep=kp)) for kp, sk in zip(keeps, LAYER_SKIP_24) if not sk)
    masked = 1.0 - sum(keeps) / (len(keeps) * w.n_tiles)
    return {
        "metric": "SSBA 24-layer stack ms/call + effective TFLOP/s (per-layer keep schedule, "
                  f"{100 * masked:.2f}% average masked, offsets alternating)",
        "value": round(gf / (ms_stack * 1e-3) / 1e12, 2), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": steps, "warmup": warmup, "ms_per_step": round(ms_stack, 5), "higher_is_better": True,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"{w.name} x 24 layers: {describe(w)} (keep per layer {list(keeps)})"},
        "clock_settle_ms": settle_ms, "clock_settle_calls": settle_calls,
        "ms_per_layer": round(ms_stack / len(keeps), 5),
        "ms_separate_fused_calls": round(ms_separate, 5),
        "ms_pruned_stack": round(ms_pruned, 5), "pruned_layers_skipped": int(sum(LAYER_SKIP_24)),
        "tflops_pruned": round(gf_pruned / (ms_pruned * 1e-3) / 1e12, 2),
        "ms_shared_gate_stack": round(ms_shared, 5),
        "ms_window_stack": round(ms_window, 5),
        "gflop_stack": round(gf / 1e9, 3),
    }


HAAR_SHAPE, HAAR_LEVELS = (4, 128, 512, 512), 3
PEAK_HBM_GBS = 8000.0


def haar_bytes(shape, levels: int, elem: int = 2):
    """Algorithmic HBM bytes: forward reads x and writes every level's four
    bands; inverse reads the coarsest LL and every level's three detail bands
    and writes the output."""
    n, c, h, w = shape
    x = n * c * h * w * elem
    lv = [n * 4 * c * (h >> l) * (w >> l) * elem for l in range(1, levels + 1)]
    fwd = x + sum(lv)
    inv = lv[-1] // 4 + sum(3 * b // 4 for b in lv) + x
    return fwd, inv


def measure_haar(steps: int, warmup: int, with_cpu: bool) -> dict:
    """The multi-level Haar transform pair of the Tiny DWT-Distilled VAE on
    four [128, 512, 512] bf16 feature maps, 3 levels (synthetic: the paper
    gives no channel count).  The 592 MiB a forward call touches exceed the
    256 MB MALL, so back-to-back calls stream from HBM."""
    import torch
    from paper_2605_15684_amd import _lib, haar
    g = torch.Generator(device="cpu").manual_seed(1)
    x = torch.randn(HAAR_SHAPE, generator=g, dtype=torch.float32).to(torch.bfloat16).to("cuda")
    lv = haar.dwt(x, HAAR_LEVELS)
    y = torch.empty_like(x)

    def span(fn, n):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(n):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    ms_dwt = span(lambda: haar.dwt(x, HAAR_LEVELS, out=lv), steps)
    ms_iwt = span(lambda: haar.iwt(lv, out=y), steps)

    # Cold single calls: a 1 GiB write before each evicts whatever part of
    # the working set the MALL still holds.
    evict = torch.empty(1 << 28, dtype=torch.float32, device="cuda")

    def cold(fn, reps=10):
        ts = []
        for r in range(reps):
            evict.fill_(float(r))
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        return sorted(ts)[reps // 2]
    ms_dwt_cold = cold(lambda: haar.dwt(x, HAAR_LEVELS, out=lv))
    ms_iwt_cold = cold(lambda: haar.iwt(lv, out=y))
    del evict
    # Reference: a plain device copy of x (read + write of 256 MiB), the
    # streaming rate a kernel can reach on this machine.
    ms_copy = span(lambda: y.copy_(x), steps)
    gbs_copy = 2 * x.numel() * x.element_size() / (ms_copy * 1e-3) / 1e9
    b_fwd, b_inv = haar_bytes(HAAR_SHAPE, HAAR_LEVELS)
    gbs_dwt = b_fwd / (ms_dwt * 1e-3) / 1e9
    gbs_iwt = b_inv / (ms_iwt * 1e-3) / 1e9
    desc = haar.haar_desc(HAAR_SHAPE, HAAR_LEVELS, torch.bfloat16)
    kernel = _lib.haar_kernel_name(desc, False)
    traffic = measured_traffic(kernel, "haar512")
    line = {
        "metric": "Haar DWT GB/s (T-DVAE multi-level Haar transform, HBM roofline)",
        "value": round(gbs_dwt, 1), "unit": "GB/s", "n_gpus": 1, "steps": steps, "warmup": warmup,
        "ms_per_step": round(ms_dwt, 5), "higher_is_better": True, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"haar512: x [4, 128, 512, 512] bf16, {HAAR_LEVELS} levels, all four bands "
                               "stored per level"},
        "ms_dwt": round(ms_dwt, 5), "ms_iwt": round(ms_iwt, 5),
        "gbs_iwt": round(gbs_iwt, 1), "bytes_dwt": b_fwd, "bytes_iwt": b_inv,
        "gbs_device_copy": round(gbs_copy, 1),
        "ms_dwt_cold": round(ms_dwt_cold, 5), "ms_iwt_cold": round(ms_iwt_cold, 5),
        "gbs_dwt_cold": round(b_fwd / (ms_dwt_cold * 1e-3) / 1e9, 1),
        "gbs_iwt_cold": round(b_inv / (ms_iwt_cold * 1e-3) / 1e9, 1),
        "roofline": {"bound": "hbm", "kernel": kernel, "achieved": round(gbs_dwt, 1), "peak": PEAK_HBM_GBS,
                     "unit": "GB/s", "frac": round(gbs_dwt / PEAK_HBM_GBS, 4),
                     "traffic": None if traffic is None else round(traffic),
                     "traffic_unit": "HBM bytes/launch", "sources_sha": sources_sha(kernel)},
        "roofline_iwt": {"bound": "hbm", "kernel": _lib.haar_kernel_name(desc, True),
                         "achieved": round(gbs_iwt, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                         "frac": round(gbs_iwt / PEAK_HBM_GBS, 4)},
    }
    if with_cpu:
        from oracle import haar_oracle as H
        xc = x[:1, :8].float().cpu().double().numpy()
        t0 = time.perf_counter()
        H.dwt(xc, HAAR_LEVELS)
        sec = time.perf_counter() - t0
        line["cpu_baseline"] = {"value": round(b_fwd / 64 / sec / 1e9, 3), "unit": "GB/s", "cores": 1,
                                "kind": "oracle",
                                "sample": f"fp64 oracle forward on 8 of 512 planes ({sec:.2f} s), pro-rated"}
    return line


def measure_backward(w, steps: int, warmup: int) -> dict:
    """Training step of one SSBA layer on the 64x64 grid: the forward with
    its log-sum-exp, then the backward (gradients of the attend step with the
    gate held fixed).  Algorithmic work: 4 D flops per computed pair in the
    forward, 10 D in the backward (dV = P^T dO, dP = dO V^T, dQ = dS K,
    dK = dS^T Q and the recomputed scores)."""
    import torch
    from paper_2605_15684_amd import _lib, ssba
    from paper_2605_15684_amd.inputs import make_qkv
    q, k, v = make_qkv(w, device="cuda")
    desc = ssba.desc_for(q, grid=(w.grid_h, w.grid_w), tile=w.tile, shift=w.shift, n_text=w.n_text,
                         gate=w.gate, keep=w.keep)
    index, _ = ssba.build_index(q, k, desc)
    out, lse = ssba.forward_train(q, k, v, index, desc)
    g = torch.Generator(device="cpu").manual_seed(w.seed + 7)
    dout = torch.randn(q.shape, generator=g, dtype=torch.float32).to(torch.bfloat16).to("cuda")
    dq, dk, dv = (torch.empty_like(q) for _ in range(3))
    sb = _lib.backward_workspace_size(desc)
    scratch = torch.empty(((sb + 7) // 8,), dtype=torch.float64, device="cuda")

    def span(fn, n):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(n):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    ms_fwd = span(lambda: ssba.forward_train(q, k, v, index, desc, out, lse), steps)
    ms_bwd = span(lambda: ssba.backward(q, k, v, out, dout, lse, index, desc, dq, dk, dv, scratch), steps)
    f_fwd = flops(w)
    f_bwd = 2.5 * f_fwd
    tf_bwd = f_bwd / (ms_bwd * 1e-3) / 1e12
    return {
        "metric": f"SSBA backward TFLOP/s (gradients of the attend step, {w.seq_len} tokens, "
                  f"{100 * (1 - pairs_per_bh(w) / w.seq_len ** 2):.0f}% sparse)",
        "value": round(tf_bwd, 2), "unit": "TFLOP/s", "n_gpus": 1, "steps": steps, "warmup": warmup,
        "ms_per_step": round(ms_bwd, 5), "higher_is_better": True, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"{w.name}: {describe(w)}"},
        "ms_forward_train": round(ms_fwd, 5), "ms_backward": round(ms_bwd, 5),
        "ms_train_step": round(ms_fwd + ms_bwd, 5),
        "tflops_train_step": round((f_fwd + f_bwd) / ((ms_fwd + ms_bwd) * 1e-3) / 1e12, 2),
        "gflop_backward": round(f_bwd / 1e9, 3),
        "roofline": {"bound": "mfma", "kernel": "k_bwd_dq + k_bwd_dkdv",
                     "achieved": round(tf_bwd, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(tf_bwd / PEAK_BF16_TFLOPS, 4)},
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--settle-ms", type=float, default=100.0,
                    help="clock-settle phase before the warm-up: back-to-back steps for this long")
    ap.add_argument("--workload", default="grid64")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--sweep", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true")
    ap.add_argument("--layers", action="store_true",
                    help="measure the 24-layer stack (ssba_forward_layers) instead of one call")
    ap.add_argument("--haar", action="store_true",
                    help="measure the multi-level Haar transform pair instead of the SSBA call")
    ap.add_argument("--backward", action="store_true",
                    help="measure the training forward and the backward of one SSBA call")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: the SSBA path runs on one GPU here "
              "(heads and batch would shard with no exchange).", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2605_15684_amd.inputs import SWEEP_TOPK_KEEP, SWEEP_WINDOW, preset
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.copy_calibration:
        src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": COPY_BYTES, "calls": 5}), flush=True)
        return

    if args.haar:
        print(json.dumps(measure_haar(args.steps, args.warmup, not args.no_cpu)), flush=True)
        return
    w = preset(args.workload)
    if args.backward:
        print(json.dumps(measure_backward(w, args.steps, args.warmup)), flush=True)
        return
    if args.layers:
        print(json.dumps(measure_layers(w, max(5, args.steps // 10), max(2, args.warmup // 10),
                                        settle_ms=args.settle_ms)), flush=True)
        return
    r, m = measure(w, args.steps, args.warmup, max(20, args.steps // 4), settle_ms=args.settle_ms)
    f = flops(w)
    from paper_2605_15684_amd import _lib

    def roofline_of(kernel, ms):
        achieved = f / (ms * 1e-3) / 1e12
        traffic = measured_traffic(kernel, w.name)
        return {"bound": "mfma", "kernel": kernel, "achieved": round(achieved, 2),
                "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                "traffic": None if traffic is None else round(traffic),
                "traffic_unit": "HBM bytes/launch", "ms_per_launch": round(ms, 5),
                "sources_sha": sources_sha(kernel)}

    ungated = roofline_of(_lib.forward_kernel(r.desc, mode=0), m["ms_fwd"])
    roofline = roofline_of(_lib.forward_kernel(r.desc, mode=2), m["ms_gated"]) if m["ms_gated"] else ungated
    mfma_meas = measured_mfma_tflops()
    cpu = None if args.no_cpu else cpu_baseline(r)
    line = {
        "metric": "SSBA fwd ms/call + effective TFLOP/s (% bf16 MFMA peak) at 4096 tokens, 84% sparse",
        "value": round(m["tflops_step"], 2), "unit": "TFLOP/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "clock_settle_ms": args.settle_ms, "clock_settle_calls": m["settle_calls"],
        "ms_per_step": round(m["ms_step"], 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"{w.name}: {describe(w)}", "global_batch": w.batch,
                   "seq_len": w.seq_len, "parallelism": "none (1 GPU)"},
        "ms_fwd": round(m["ms_fwd"], 5), "ms_index": round(m["ms_index"], 5),
        "ms_gated": None if m["ms_gated"] is None else round(m["ms_gated"], 5),
        "ms_pool": None if m["ms_pool"] is None else round(m["ms_pool"], 5),
        "ms_step_rope": None if m["ms_step_rope"] is None else round(m["ms_step_rope"], 5),
        "ms_rope_pool": None if m["ms_rope_pool"] is None else round(m["ms_rope_pool"], 5),
        "gbs_rope_pool": None if m["ms_rope_pool"] is None else round(rope_bytes(w) / (m["ms_rope_pool"] * 1e-3) / 1e9, 1),
        "ms_dense": round(m["ms_dense"], 5), "ms_step_wall": round(m["ms_step_wall"], 5),
        "ms_step_eager": round(m["ms_step_eager"], 5),
        "ms_step_two_calls": round(m["ms_step_two_calls"], 5),
        "ms_step_cold": round(m["ms_step_cold"], 5), "ms_fwd_cold": round(m["ms_fwd_cold"], 5),
        "ms_step_graph": None if m["ms_step_graph"] is None else round(m["ms_step_graph"], 5),
        "tflops_fwd": round(m["tflops_fwd"], 2), "pct_peak_fwd": round(100 * m["tflops_fwd"] / PEAK_BF16_TFLOPS, 2),
        "mfma_measured_tflops": round(mfma_meas, 1),
        "pct_measured_peak_fwd": round(100 * m["tflops_fwd"] / mfma_meas, 2),
        "tflops_dense": round(m["tflops_dense"], 2),
        "speedup_vs_dense_kernel": round(m["speedup_kernel"], 3),
        "speedup_vs_dense_step": round(m["speedup_step"], 3),
        "gflop_computed": round(m["gflop"], 3), "gflop_dense": round(m["gflop_dense"], 3),
        "roofline": roofline, "roofline_ungated": ungated, "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)

    if args.sweep:
        cases = [preset("sweep64", keep=kp) for kp in SWEEP_TOPK_KEEP.values()]
        cases += [preset("sweep64", gate="window", window=wd) for wd in SWEEP_WINDOW.values()]
        cases += [preset("grid64_text"), preset("grid128")]
        for c in cases:
            del r
            torch.cuda.empty_cache()
            r, mm = measure(c, max(20, args.steps // 2), args.warmup, 20, graph=False, settle_ms=args.settle_ms)
            print(json.dumps({"workload": c.name, "desc": describe(c),
                              **{k: (None if v is None else round(v, 5)) for k, v in mm.items()},
                              "pct_peak_fwd": round(100 * mm["tflops_fwd"] / PEAK_BF16_TFLOPS, 2)}),
                  file=sys.stderr, flush=True)


if __name__ == "__main__":
    main()
