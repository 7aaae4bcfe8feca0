#!/usr/bin/env python3
"""Packed-KV decode benchmark on one MI355X.

Headline workload (Llama-3.1-8B-shaped full decode step): 32 layers, 32 query
heads, 8 KV heads (G = 4), d_h = 128, RoPE base 5e5, bf16 inputs, batch 1,
128K cached rows, K2V2 (B = 128, b_V = 2), per-(layer, head) widths from the
greedy allocator on 2048 synthetic calibration tokens.  One step appends and
quantizes one row for every (layer, KV head) and then runs the split-context
decode attention of every layer over the packed cache (one all-layer launch
of each entry point).  Inputs are resident in HBM before timing starts.

Before the timed loop an untimed settle phase repeats the step for a fixed
wall time (reported), so that the timed steps start with the device clock in
its steady state, whatever the number of warm-up steps.  Ratios against
comparators come from interleaved A/B loops (one call of each per round).

The other workloads of the measurement plan are reported beside it (each its
own sub-object): the toy single head, one Qwen2.5-3B-shaped layer at 32K (the
prefill call and the median of 64 steps), the Qwen2.5-3B-shaped K3V3 step at
128K / 256K / 512K rows (with the fp16 comparator and packed-vs-fp16 bytes),
the ragged batch of 8 (cold and warm; the toy head and the 32K layer are
also timed cold, after a 1 GiB cache flush per step), the prefill
quantize_append against the fp32 roofline, a read-probe ceiling, the
headline step as per-layer launches replayed from a HIP graph, and the fp64
CPU oracle on the host's cores (with the headline's parity statistics).

Prints one JSON line.  The design notes give the roofline definitions.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
FP32_PEAK_TFLOPS = 157.3
F16_MFMA_PEAK_TFLOPS = 2500.0
KERNEL_SRC = os.path.join(ROOT, "paper_2606_24033_amd", "csrc", "decode_impl.h")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "k_split_mfma_llama8b_128k_k2v2_traffic.json")
N_SINK, N_RECENT = 4, 128      # protected-buffer regime of the reasoning evaluation
N_CAL = 2048

LLAMA = dict(name="Llama-3.1-8B", seed=3, n_layers=32, n_kv=8, group=4, base=5e5, k_budget=128, v_bits=2)
QWEN_LONG = dict(name="Qwen2.5-3B", seed=5, n_layers=36, n_kv=2, group=8, base=1e6, k_budget=192, v_bits=3)


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=30)
    ap.add_argument("--ctx", type=int, default=131072)
    ap.add_argument("--n-splits", type=int, default=0)
    ap.add_argument("--settle-s", type=float, default=2.0,
                    help="untimed settle phase before the timed loop (wall seconds of repeated steps)")
    ap.add_argument("--no-fp16", action="store_true", help="skip the fp16 comparator")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-prefill", action="store_true",
                    help="skip the prefill-attention measurement (one layer, 32K-token prompt)")
    ap.add_argument("--prefill-len", type=int, default=32768)
    ap.add_argument("--no-uniform", action="store_true",
                    help="skip the uniform TQ-MSE K layout (one K group per head) comparison")
    ap.add_argument("--no-protected", action="store_true",
                    help="skip the protected fp16 window (4 sink + 128 recent rows) measurement")
    ap.add_argument("--no-rope-step", action="store_true",
                    help="skip the pre-RoPE step measurement (eager and graph-replayed)")
    ap.add_argument("--no-workloads", action="store_true",
                    help="skip the other workloads (toy, Qwen-shaped 32K layer / 128K / 256K / 512K, ragged batch)")
    ap.add_argument("--no-long", action="store_true", help="skip the 256K and 512K Qwen-shaped steps")
    ap.add_argument("--only-headline", action="store_true", help="the headline step and its roofline only")
    ap.add_argument("--model", choices=["llama8b_k2v2", "qwen3b_k3v3"], default="llama8b_k2v2",
                    help="workload of the headline step (qwen3b_k3v3: 36 layers x 2 KV heads, G = 8, K3V3, "
                         "8192-row prefill chunks; for profiles with --only-headline)")
    ap.add_argument("--cpu-workers", type=int, default=0, help="CPU baseline processes (0: host CPUs, at most 16)")
    ap.add_argument("--copy-calib-mib", type=int, default=0,
                    help="run one plain device copy of this size first (HBM counter calibration)")
    return ap.parse_args()


def kernel_sha():
    with open(KERNEL_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def measured_traffic():
    """HBM bytes per decode launch from the committed counter summary, or None
    when the decode kernel source changed after the counters were taken."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("kernel_src_sha256") != kernel_sha():
        return None
    return t.get("traffic_bytes_per_launch")


def stats(us):
    a = np.asarray(us, dtype=np.float64)
    return {"median": round(float(np.median(a)), 2), "mean": round(float(a.mean()), 2),
            "p5": round(float(np.percentile(a, 5)), 2), "p95": round(float(np.percentile(a, 95)), 2), "n": int(a.size)}


def ev_pair(torch):
    return torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)


def settle(torch, fn, seconds):
    """Repeat fn (untimed) for `seconds` of wall time; returns what was done."""
    if seconds <= 0:
        return {"seconds": 0.0, "calls": 0}
    t0 = time.perf_counter()
    n = 0
    while True:
        for _ in range(8):
            fn()
            n += 1
        torch.cuda.synchronize()
        if time.perf_counter() - t0 >= seconds:
            break
    return {"seconds": round(time.perf_counter() - t0, 3), "calls": n}


def interleaved(torch, fns, n):
    """n rounds; in round i every fn(i) runs once between HIP events on the
    current stream (the stream the library launches on).  Per-fn µs lists."""
    evs = [[ev_pair(torch) for _ in range(n)] for _ in fns]
    for i in range(n):
        for j, f in enumerate(fns):
            evs[j][i][0].record()
            f(i)
            evs[j][i][1].record()
    torch.cuda.synchronize()
    return [[a.elapsed_time(b) * 1e3 for a, b in e] for e in evs]


def n_groups(bits):
    return np.array([[len(np.unique(bits[layer, h])) for h in range(bits.shape[1])] for layer in range(bits.shape[0])])


def quantize_flops_per_row(bits_row):
    """Algorithmic fp32 flops of encoding one key row and one value row: the
    group rotations (2 d_g^2 each) and the value rotation (2 d_h^2)."""
    dg = [2 * int(np.sum(bits_row == b)) for b in range(1, 9)]
    return 2.0 * (sum(d * d for d in dg) + 128 * 128)


class Model:
    """One synthetic model-shaped decode workload over the packed cache
    (batch 1): widths from the library's allocator on calibration data,
    the prompt quantized into the cache (in chunks if asked), then per step
    one appended row and one all-layer decode."""

    def __init__(self, bg, synth, torch, spec, T, n_steps, *, chunk=None, fp16=False, window=False,
                 in_dtype=None, n_cal=N_CAL, n_splits=0):
        self.bg, self.synth, self.torch = bg, synth, torch
        self.spec, self.T, self.n_steps = spec, T, n_steps
        self.L, self.H, self.G = spec["n_layers"], spec["n_kv"], spec["group"]
        self.seed, self.base = spec["seed"], spec["base"]
        self.kb, self.vb = spec["k_budget"], spec["v_bits"]
        self.n_splits = n_splits
        self.in_dtype = bg.BGTQ_BF16 if in_dtype is None else in_dtype
        tdt = torch.bfloat16 if self.in_dtype == bg.BGTQ_BF16 else torch.float32
        self.max_ctx = T + n_steps
        cap = ((T + n_steps + 63) // 64) * 64
        self.cfg = bg.Config(n_layers=self.L, batch=1, n_kv_heads=self.H, group=self.G, capacity=cap,
                             k_budget=self.kb, v_bits=self.vb, in_dtype=self.in_dtype)
        self.bits = np.zeros((self.L, self.H, 64), np.uint8)
        self.sig = np.zeros((self.L, self.H, 64))
        for layer in range(self.L):
            for h in range(self.H):
                self.sig[layer, h] = synth.sigma_profile(self.seed, layer, h)
                qc, kc = synth.calibration(self.seed, layer, h, n_cal, self.G, self.sig[layer, h])
                s = bg.blockgtq_energy_scores(qc.astype(np.float32), kc.astype(np.float32))
                self.bits[layer, h] = bg.blockgtq_allocate(s, self.kb)[0]
        self.rot_k, self.rot_v = synth.rotations(self.seed)
        self.layout = bg.Layout(self.cfg, self.bits, synth.flat_rot_k(self.rot_k), self.rot_v)
        self.cache = bg.Cache(self.cfg)
        if fp16:
            self.k16 = torch.zeros((self.L, 1, self.H, cap, 128), dtype=torch.float16, device="cuda")
            self.v16 = torch.zeros_like(self.k16)
        self.window = None
        if window:
            self.window = torch.zeros(bg.window_bytes(self.cfg, N_SINK, N_RECENT) // 2, dtype=torch.float16,
                                      device="cuda")
        self.knew = torch.empty((n_steps, self.L, 1, 1, self.H, 128), dtype=tdt, device="cuda")
        self.vnew = torch.empty_like(self.knew)
        self.prefill_us = []
        chunk = T if chunk is None else chunk
        for layer in range(self.L):
            k, v = synth.torch_layer_kv(self.seed, layer, T + n_steps, self.sig[layer], self.base, dtype=tdt)
            for c0 in range(0, T, chunk):
                n = min(chunk, T - c0)
                kk, vv = k[None, c0:c0 + n].contiguous(), v[None, c0:c0 + n].contiguous()
                wp = torch.tensor([c0], dtype=torch.int32, device="cuda")
                a, b = ev_pair(torch)
                a.record()
                bg.blockgtq_quantize_append(self.cfg, self.layout, layer, kk, vv, wp, self.cache)
                b.record()
                self.prefill_us.append((a, b, n))
                if window:
                    bg.blockgtq_window_append(self.cfg, layer, kk, vv, wp, N_SINK, N_RECENT, self.window)
            if fp16:
                self.k16[layer, 0, :, :T + n_steps] = k.transpose(0, 1).half()
                self.v16[layer, 0, :, :T + n_steps] = v.transpose(0, 1).half()
            self.knew[:, layer, 0, 0] = k[T:]
            self.vnew[:, layer, 0, 0] = v[T:]
            del k, v
        torch.cuda.synchronize()
        self.prefill_us = [(a.elapsed_time(b) * 1e3, n) for a, b, n in self.prefill_us]
        positions = list(range(T, T + n_steps))
        self.q = torch.stack([synth.torch_queries(self.seed, layer, self.H * self.G, positions, self.base, dtype=tdt)
                              for layer in range(self.L)], dim=1)[:, :, None].contiguous()  # [steps, L, 1, Hq, 128]
        self.wps = torch.arange(T, T + n_steps, dtype=torch.int32, device="cuda")
        self.ctxs = self.wps + 1
        self.out = torch.empty((self.L, 1, self.H * self.G, 128), dtype=torch.float32, device="cuda")
        self.ws = torch.zeros(bg.workspace_bytes(self.cfg, self.L, n_splits, self.max_ctx), dtype=torch.uint8,
                              device="cuda")
        self.ng = n_groups(self.bits)

    # ---- one step = append one row everywhere, then decode every layer
    def append(self, s):
        self.bg.blockgtq_quantize_append(self.cfg, self.layout, -1, self.knew[s], self.vnew[s], self.wps[s:s + 1],
                                         self.cache)

    def decode(self, s):
        self.bg.blockgtq_decode_attn(self.cfg, self.layout, -1, self.q[s], self.ctxs[s:s + 1], self.max_ctx,
                                     self.cache, out=self.out, workspace=self.ws, n_splits=self.n_splits)

    def decode_fp16(self, s, out):
        self.bg.blockgtq_decode_attn_fp16(self.cfg, -1, self.q[s], self.ctxs[s:s + 1], self.max_ctx, self.k16,
                                          self.v16, out=out, workspace=self.ws, n_splits=self.n_splits)

    def step(self, s):
        self.append(s)
        self.decode(s)

    def row_bytes(self):
        """Algorithmic bytes of one row summed over every (layer, KV head):
        codes 128 (b_K + b_V) / 8, 2 n_g bytes of K radii, 2 of the V radius."""
        codes = (2 * self.kb / 8 + 128 * self.vb / 8 + 2) * self.L * self.H
        return codes + 2.0 * self.ng.sum()

    def io_bytes(self):
        qb = 2 if self.in_dtype == self.bg.BGTQ_BF16 else 4
        return self.L * self.H * self.G * 128 * (qb + 4)

    def step_bytes(self, ctx):
        return ctx * self.row_bytes() + self.io_bytes()

    def fp16_bytes(self, ctx):
        return ctx * self.L * self.H * 512.0

    def cache_bytes_used(self, rows):
        """Allocated packed-cache bytes holding `rows` rows (codes, radii at
        their token-major stride, value radii) against fp16 K/V."""
        per_row = self.cfg.k_words * 4 + 128 * self.vb / 8 + 2
        radii = 2.0 * sum(int(g + (g & 1)) for g in self.ng.reshape(-1))
        packed = rows * (per_row * self.L * self.H + radii)
        return int(packed), int(rows * self.L * self.H * 512)

    def free(self):
        for name in ("cache", "layout", "k16", "v16", "window", "knew", "vnew", "q", "out", "ws"):
            if hasattr(self, name):
                delattr(self, name)
        self.torch.cuda.empty_cache()


def timed_steps(torch, m, first, n):
    """Steps first .. first+n-1 with events around the loop and around each
    decode launch (every event is a marker that the stream waits on, a few µs
    each, so the steps carry no others); step i runs from the end of decode
    i - 1 (the loop's start for i = 0) to the end of decode i.  Returns
    (step µs, decode µs, total ms on events)."""
    evd = [ev_pair(torch) for _ in range(n)]
    g0, g1 = ev_pair(torch)
    torch.cuda.synchronize()
    g0.record()
    for i in range(n):
        s = first + i
        m.append(s)
        evd[i][0].record()
        m.decode(s)
        evd[i][1].record()
    g1.record()
    torch.cuda.synchronize()
    starts = [g0] + [evd[i][1] for i in range(n - 1)]
    return ([a.elapsed_time(evd[i][1]) * 1e3 for i, a in enumerate(starts)],
            [a.elapsed_time(b) * 1e3 for a, b in evd], g0.elapsed_time(g1))


def sdpa_decode_context(torch, m, W, K):
    """Context for the fp16 comparator: torch's scaled_dot_product_attention
    (fp16, one query row per head, grouped KV heads) over the same fp16 cache,
    all layers in one call (layers as the batch).  None if torch refuses."""
    try:
        sdpa = torch.nn.functional.scaled_dot_product_attention
        ctx = int(m.ctxs[W].item())
        k = m.k16[:, 0, :, :ctx]
        v = m.v16[:, 0, :, :ctx]
        qs = [m.q[W + i][:, 0].half()[:, :, None] for i in range(min(K, 8))]
        fn = lambda i: sdpa(qs[i % len(qs)], k, v, enable_gqa=True)
        fn(0)
        torch.cuda.synchronize()
        us = interleaved(torch, [fn], K)[0]
        byt = m.fp16_bytes(ctx) + m.io_bytes()
        return {"call_us": stats(us), "gbs": round(byt / (np.median(us) * 1e-6) / 1e9, 2),
                "pct_hbm_peak": round(100 * byt / (np.median(us) * 1e-6) / 1e9 / HBM_PEAK_GBS, 2),
                "note": "torch fp16 SDPA, q_len 1, enable_gqa, layers as the batch; context only"}
    except Exception as e:  # noqa: BLE001 - context only
        log(f"torch SDPA decode context unavailable: {e}")
        return None


def cold_warm_steps(torch, m, first, n, flush_bytes=1 << 30):
    """Steps first .. first+n-1 again (the same rows at the same positions:
    the cache content does not change), each twice in a row and timed alike:
    warm, then after an untimed write of a 1 GiB buffer that evicts the L2
    and MALL (cold: the step from HBM)."""
    flush = torch.empty(flush_bytes, dtype=torch.uint8, device="cuda")
    evw = [ev_pair(torch) for _ in range(n)]
    evc = [ev_pair(torch) for _ in range(n)]
    for i in range(n):
        evw[i][0].record()
        m.step(first + i)
        evw[i][1].record()
        flush.fill_(i & 255)
        evc[i][0].record()
        m.step(first + i)
        evc[i][1].record()
    torch.cuda.synchronize()
    del flush
    return [a.elapsed_time(b) * 1e3 for a, b in evw], [a.elapsed_time(b) * 1e3 for a, b in evc]


def workload_line(torch, m, args, label, settle_s, fp16=False, cold=False):
    """Settle, K timed steps, then (cold) the same steps after a cache flush
    each, then (fp16) the packed and fp16 decodes interleaved at the timed
    steps' contexts."""
    W = min(args.warmup, m.n_steps - args.steps)
    for s in range(W):
        m.step(s)
    st = settle(torch, lambda: m.step(W), settle_s)
    step_us, dec_us, total_ms = timed_steps(torch, m, W, args.steps)
    ctx_mean = m.T + W + (args.steps + 1) / 2.0
    sb = m.step_bytes(ctx_mean)
    dmean = float(np.mean(dec_us))
    packed, f16b = m.cache_bytes_used(m.T + m.n_steps)
    res = {"workload": label, "ctx": m.T, "settle": st, "step_us": stats(step_us), "decode_us": stats(dec_us),
           "ms_per_step": round(total_ms / args.steps, 4),
           "algorithmic_bytes_per_step": int(sb),
           "step_gbs": round(sb / (total_ms / args.steps * 1e-3) / 1e9, 2),
           "roofline": {"bound": "hbm", "achieved": round(sb / (dmean * 1e-6) / 1e9, 2), "peak": HBM_PEAK_GBS,
                        "unit": "GB/s", "frac": round(sb / (dmean * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
                        "kernel": "k_split_mfma", "launch_us_mean": round(dmean, 2)},
           "cache_bytes": {"packed": packed, "fp16": f16b, "compression": round(f16b / packed, 3)},
           "prefill_quantize_us": stats([u for u, _ in m.prefill_us]),
           "prefill_rows_per_call": int(m.prefill_us[0][1] * m.H)}
    if cold:
        wu, cu = cold_warm_steps(torch, m, W, args.steps)
        res["flush_ab"] = {"warm_step_us": stats(wu), "cold_step_us": stats(cu),
                           "cold_step_gbs": round(sb / (np.median(cu) * 1e-6) / 1e9, 2),
                           "note": "each step timed twice alike: warm, then after a 1 GiB flush"}
    if fp16:
        out16 = torch.empty_like(m.out)
        p_us, f_us = interleaved(torch, [lambda i: m.decode(W + i), lambda i: m.decode_fp16(W + i, out16)],
                                 args.steps)
        fb = m.fp16_bytes(ctx_mean) + m.io_bytes()
        res["fp16_comparator"] = {
            "kernel": "k_f16_mfma", "decode_us": stats(f_us), "packed_decode_us_interleaved": stats(p_us),
            "gbs": round(fb / (np.mean(f_us) * 1e-6) / 1e9, 2),
            "pct_hbm_peak": round(100 * fb / (np.mean(f_us) * 1e-6) / 1e9 / HBM_PEAK_GBS, 2),
            "speedup_packed_over_fp16": round(float(np.median(f_us) / np.median(p_us)), 3)}
        sd = sdpa_decode_context(torch, m, W, args.steps)
        if sd is not None:
            res["fp16_comparator"]["torch_sdpa_fp16_decode"] = sd
    return res


# ------------------------------------------------------------------ legs

def uniform_comparison(bg, synth, torch, m, args, W):
    """The same decode over a uniform TQ-MSE K layout: every RoPE block at
    k_budget / 64 bits, i.e. one K group of 128 coordinates and one K radius
    per row (the paper's uniform-TQ-MSE baseline, which differs from Block-GTQ
    only in the K layout), interleaved with the Block-GTQ decode at the timed
    steps' contexts over a cache prefilled with all their rows."""
    ubits = np.full((m.L, m.H, 64), m.kb // 64, np.uint8)
    ulayout = bg.Layout(m.cfg, ubits, synth.flat_rot_k(m.rot_k), m.rot_v)
    ucache = bg.Cache(m.cfg)
    wp0 = torch.zeros(1, dtype=torch.int32, device="cuda")
    for layer in range(m.L):
        k, v = synth.torch_layer_kv(m.seed, layer, m.T + m.n_steps, m.sig[layer], m.base)
        bg.blockgtq_quantize_append(m.cfg, ulayout, layer, k[None].contiguous(), v[None].contiguous(), wp0, ucache)
        del k, v
    uout = torch.empty_like(m.out)

    def udec(i):
        s = W + i
        bg.blockgtq_decode_attn(m.cfg, ulayout, -1, m.q[s], m.ctxs[s:s + 1], m.max_ctx, ucache, out=uout,
                                workspace=m.ws, n_splits=m.n_splits)

    for i in range(3):
        udec(i)
    b_us, u_us = interleaved(torch, [lambda i: m.decode(W + i), udec], args.steps)
    ctx_mean = m.T + W + (args.steps + 1) / 2.0
    ubytes = ctx_mean * m.L * m.H * (m.kb * 2 / 8 + 2 + 128 * m.vb / 8 + 2) + m.io_bytes()
    res = {"decode_us": stats(u_us), "block_gtq_decode_us_interleaved": stats(b_us), "bytes_per_call": int(ubytes),
           "gbs": round(ubytes / (np.mean(u_us) * 1e-6) / 1e9, 2),
           "pct_hbm_peak": round(100 * ubytes / (np.mean(u_us) * 1e-6) / 1e9 / HBM_PEAK_GBS, 2),
           "block_gtq_time_over_uniform": round(float(np.median(b_us) / np.median(u_us)), 3)}
    del ucache, ulayout
    torch.cuda.empty_cache()
    return res


def protected_measurement(bg, torch, m, args, W):
    """The same decode in the protected-buffer regime: the first N_SINK and the
    last N_RECENT rows of every (layer, KV head) served from an fp16 window
    (blockgtq_decode_attn_protected: the window kernel, then the packed decode
    over the rows in between), interleaved with the no-buffer decode at the
    timed steps' contexts.  The window holds the step rows too (appended after
    the timed loop, so the ring holds the last context's recent rows)."""
    for s in range(m.n_steps):
        bg.blockgtq_window_append(m.cfg, -1, m.knew[s], m.vnew[s], m.wps[s:s + 1], N_SINK, N_RECENT, m.window)
    wout = torch.empty_like(m.out)
    wws = torch.zeros(bg.protected_workspace_bytes(m.cfg, m.L, m.n_splits, m.max_ctx), dtype=torch.uint8,
                      device="cuda")

    def prot(i):
        s = W + i
        bg.blockgtq_decode_attn_protected(m.cfg, m.layout, -1, m.q[s], m.ctxs[s:s + 1], m.max_ctx, m.cache,
                                          m.window, N_SINK, N_RECENT, out=wout, workspace=wws, n_splits=m.n_splits)

    for i in range(3):
        prot(i)
    d_us, p_us = interleaved(torch, [lambda i: m.decode(W + i), prot], args.steps)
    return {"n_sink": N_SINK, "n_recent": N_RECENT, "decode_us": stats(p_us),
            "no_buffer_decode_us_interleaved": stats(d_us),
            "time_over_no_buffer": round(float(np.median(p_us) / np.median(d_us)), 3),
            "kernels": "k_window_attn + k_split_mfma (packed rows between the windows)"}


def rope_step_measurement(bg, torch, m, args, W):
    """The decode step from pre-RoPE inputs (blockgtq_rope_decode_step: RoPE on
    the device, then the all-layer append and decode), eager and as a captured
    graph replayed with the position copied into the captured buffer before
    each replay, interleaved with the post-RoPE step.  Runs after the other
    legs and rewrites the step rows."""
    ws = torch.zeros(bg.rope_step_workspace_bytes(m.cfg, m.max_ctx, m.n_splits), dtype=torch.uint8, device="cuda")
    out = torch.empty_like(m.out)

    def eager(s):
        bg.blockgtq_rope_decode_step(m.cfg, m.layout, m.base, m.q[s], m.knew[s], m.vnew[s], m.wps[s:s + 1],
                                     m.max_ctx, m.cache, out=out, workspace=ws, n_splits=m.n_splits)

    q_in, k_in, v_in = m.q[0].clone(), m.knew[0].clone(), m.vnew[0].clone()
    pos = m.wps[W:W + 1].clone()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        with torch.cuda.graph(graph, stream=side):
            bg.blockgtq_rope_decode_step(m.cfg, m.layout, m.base, q_in, k_in, v_in, pos, m.max_ctx, m.cache,
                                         out=out, workspace=ws, n_splits=m.n_splits, stream=side)
    torch.cuda.synchronize()

    def replay(i):
        s = W + i
        pos.copy_(m.wps[s:s + 1])
        graph.replay()

    for i in range(max(3, min(args.warmup, 10))):  # the first replays also upload the graph
        replay(i % args.steps)
        eager(W + i % args.steps)
    torch.cuda.synchronize()
    p_us, e_us, g_us = interleaved(torch, [lambda i: m.step(W + i), lambda i: eager(W + i), replay], args.steps)
    del graph
    return {"post_rope_step_us_interleaved": stats(p_us), "eager_us": stats(e_us), "graph_us": stats(g_us),
            "eager_over_post_rope_step": round(float(np.median(e_us) / np.median(p_us)), 3),
            "graph_over_post_rope_step": round(float(np.median(g_us) / np.median(p_us)), 3),
            "kernels": "k_rope_step + k_append_rows + k_split_mfma"}


def per_layer_graph_measurement(bg, torch, m, args, W):
    """The headline step as per-layer launches: for every layer its append and
    its decode (2 x 32 launches) captured in one HIP graph, replayed with the
    step's rows, queries and position copied into the captured buffers before
    each replay, interleaved with the all-layer step (two launches)."""
    ws1 = torch.zeros(bg.workspace_bytes(m.cfg, 1, m.n_splits, m.max_ctx), dtype=torch.uint8, device="cuda")
    k_in, v_in, q_in = m.knew[W].clone(), m.vnew[W].clone(), m.q[W].clone()
    wp, cx = m.wps[W:W + 1].clone(), m.ctxs[W:W + 1].clone()
    out = torch.empty_like(m.out)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        with torch.cuda.graph(graph, stream=side):
            for layer in range(m.L):
                bg.blockgtq_quantize_append(m.cfg, m.layout, layer, k_in[layer], v_in[layer], wp, m.cache,
                                            stream=side)
                bg.blockgtq_decode_attn(m.cfg, m.layout, layer, q_in[layer], cx, m.max_ctx, m.cache, out=out[layer],
                                        workspace=ws1, n_splits=m.n_splits, stream=side)
    torch.cuda.synchronize()

    def replay(i):
        s = W + i
        k_in.copy_(m.knew[s])
        v_in.copy_(m.vnew[s])
        q_in.copy_(m.q[s])
        wp.copy_(m.wps[s:s + 1])
        cx.copy_(m.ctxs[s:s + 1])
        graph.replay()

    for i in range(max(3, min(args.warmup, 10))):  # the first replays also upload the graph
        replay(i % args.steps)
        m.step(W + i % args.steps)
    torch.cuda.synchronize()
    a_us, g_us = interleaved(torch, [lambda i: m.step(W + i), replay], args.steps)
    torch.cuda.synchronize()
    # the last round's outputs of the two forms (same step; the split plans differ)
    diff = float(((out - m.out).abs().max() / m.out.abs().max()).item())
    del graph
    return {"all_layer_step_us_interleaved": stats(a_us), "per_layer_graph_step_us": stats(g_us),
            "max_rel_diff_vs_all_layer_step": round(diff, 7),
            "graph_over_all_layer_step": round(float(np.median(g_us) / np.median(a_us)), 3),
            "launches": f"graph: {2 * m.L} (append + decode per layer) and 5 input copies; all-layer step: 2"}


def prefill_measurement(bg, synth, torch, m, T):
    """Causal prefill attention over the packed cache for one layer of the same
    model shape: a T-token prompt quantized into a one-layer cache (layer 0's
    widths), then blockgtq_prefill_attn for all T query positions.  Timed with
    HIP events; torch's fp16 causal scaled_dot_product_attention over the same
    (unquantized) K/V is timed beside it for context."""
    cfg = bg.Config(n_layers=1, batch=1, n_kv_heads=m.H, group=m.G, capacity=((T + 63) // 64) * 64,
                    k_budget=m.kb, v_bits=m.vb, in_dtype=bg.BGTQ_BF16)
    layout = bg.Layout(cfg, m.bits[:1], synth.flat_rot_k(m.rot_k), m.rot_v)
    cache = bg.Cache(cfg)
    k, v = synth.torch_layer_kv(m.seed, 0, T, m.sig[0], m.base)
    bg.blockgtq_quantize_append(cfg, layout, 0, k[None].contiguous(), v[None].contiguous(),
                                torch.zeros(1, dtype=torch.int32, device="cuda"), cache)
    q = synth.torch_queries(m.seed, 0, m.H * m.G, list(range(T)), m.base).reshape(1, T, m.H * m.G, 128).contiguous()
    qp = torch.zeros(1, dtype=torch.int32, device="cuda")
    out = torch.empty((1, T, m.H * m.G, 128), dtype=torch.float32, device="cuda")
    ws = torch.empty(bg.prefill_workspace_bytes(cfg, T), dtype=torch.uint8, device="cuda")

    def timed(fn, n=5, warm=2):
        for _ in range(warm):
            fn()
        torch.cuda.synchronize()
        ev = [ev_pair(torch) for _ in range(n)]
        for a, b in ev:
            a.record()
            fn()
            b.record()
        torch.cuda.synchronize()
        return float(np.median([a.elapsed_time(b) for a, b in ev]))

    ms = timed(lambda: bg.blockgtq_prefill_attn(cfg, layout, 0, q, qp, T - 1, cache, out=out, workspace=ws))
    flops = m.H * m.G * (T * (T + 1) / 2) * 2 * (128 + 128)
    res = {"workload": f"one {m.spec['name']}-shaped layer ({m.H} KV heads, {m.H * m.G} q heads), {T}-token "
                       f"prompt, causal, K{m.kb // 64}V{m.vb}",
           "ms_per_call": round(ms, 3), "algorithmic_tflops": round(flops / ms / 1e9, 1),
           "roofline": {"bound": "mfma", "achieved": round(flops / ms / 1e9, 1), "peak": F16_MFMA_PEAK_TFLOPS,
                        "unit": "TFLOP/s", "frac": round(flops / ms / 1e9 / F16_MFMA_PEAK_TFLOPS, 4),
                        "flops_per_call": flops, "kernel": "k_prefill_qrot + k_prefill_attn"}}
    try:
        k16 = k.half().transpose(0, 1)[None].repeat_interleave(m.G, dim=1).contiguous()
        v16 = v.half().transpose(0, 1)[None].repeat_interleave(m.G, dim=1).contiguous()
        q16 = q.half().transpose(1, 2).contiguous()
        sdpa = torch.nn.functional.scaled_dot_product_attention
        ms16 = timed(lambda: sdpa(q16, k16, v16, is_causal=True))
        res["torch_sdpa_fp16_causal_ms"] = round(ms16, 3)
        res["packed_over_fp16_time"] = round(ms / ms16, 3)
        del k16, v16, q16
    except Exception as e:  # pragma: no cover - comparator only
        log(f"fp16 SDPA comparator unavailable: {e}")
    del cache, layout, out, ws, q, k, v
    torch.cuda.empty_cache()
    return res


def quantize_roofline(m, label):
    """The prefill quantize_append calls of a workload's setup (one call per
    layer and chunk, HIP events) against the fp32 MFMA peak: algorithmic flops
    per row = the group rotations and the value rotation."""
    us = np.array([u for u, _ in m.prefill_us])
    rows_per_call = m.prefill_us[0][1]
    fl_head = np.mean([[quantize_flops_per_row(m.bits[layer, h]) for h in range(m.H)] for layer in range(m.L)],
                      axis=0).sum()                     # flops of one row of every head of a layer
    mean_us = float(us.mean())
    tfl = rows_per_call * fl_head / (mean_us * 1e-6) / 1e12
    return {"workload": label, "rows_per_call": int(rows_per_call * m.H), "calls": int(us.size),
            "call_us": stats(us), "rows_per_s": round(rows_per_call * m.H / (mean_us * 1e-6), 1),
            "flops_per_row": round(fl_head / m.H, 1),
            "roofline": {"bound": "mfma", "achieved": round(tfl, 2), "peak": FP32_PEAK_TFLOPS, "unit": "TFLOP/s",
                         "frac": round(tfl / FP32_PEAK_TFLOPS, 4), "kernel": "k_quant_rows"}}


def ragged_workload(bg, synth, torch, args, flush_bytes=1 << 30):
    """Ragged batched decode: Llama-3.1-8B attention shape (1 layer, 8 KV
    heads, G = 4, base 5e5, bf16), batch 8 with contexts drawn uniformly from
    [4096, 65536], K3V2.  Each step appends one row per sequence at its own
    position and decodes; per-step time warm (steps back to back; the
    ~0.2 GB working set can stay in the 256 MB MALL) and cold (a 1 GiB buffer
    written between steps, untimed).  Plus one 16384-row prefill call for the
    whole batch."""
    seed, L, B, H, G, base, kb, vb = 4, 1, 8, 8, 4, 5e5, 192, 2
    ctx = [int(x) for x in synth.ragged_lengths(seed, B, 4096, 65536)]
    n_steps = 2 * args.steps + 4
    Tm = max(max(ctx) + n_steps, 16384)
    cfg = bg.Config(n_layers=L, batch=B, n_kv_heads=H, group=G, capacity=((Tm + 63) // 64) * 64, k_budget=kb,
                    v_bits=vb, in_dtype=bg.BGTQ_BF16)
    bits = np.zeros((L, H, 64), np.uint8)
    sig = np.zeros((H, 64))
    for h in range(H):
        sig[h] = synth.sigma_profile(seed, 0, h)
        qc, kc = synth.calibration(seed, 0, h, N_CAL, G, sig[h])
        bits[0, h] = bg.blockgtq_allocate(bg.blockgtq_energy_scores(qc.astype(np.float32), kc.astype(np.float32)),
                                          kb)[0]
    rot_k, rot_v = synth.rotations(seed)
    layout = bg.Layout(cfg, bits, synth.flat_rot_k(rot_k), rot_v)
    cache = bg.Cache(cfg)
    chunk = 16384
    # every sequence gets at least a chunk of rows: the timed 16384-row prefill
    # call writes them all (rows past a context are never attended)
    kv = [synth.torch_layer_kv(seed * 16 + b, 0, max(ctx[b] + n_steps, chunk), sig, base) for b in range(B)]
    # one 16384-row prefill call for the batch (timed), then the rest of each context
    K = torch.stack([k[:chunk] for k, _ in kv]).contiguous()
    V = torch.stack([v[:chunk] for _, v in kv]).contiguous()
    wp0 = torch.zeros(B, dtype=torch.int32, device="cuda")
    for _ in range(2):
        bg.blockgtq_quantize_append(cfg, layout, 0, K, V, wp0, cache)
    pre_us = interleaved(torch, [lambda i: bg.blockgtq_quantize_append(cfg, layout, 0, K, V, wp0, cache)], 5)[0]
    del K, V
    for c0 in range(chunk, max(ctx), chunk):
        n = min(chunk, max(ctx) - c0)
        K = torch.zeros((B, n, H, 128), dtype=torch.bfloat16, device="cuda")
        V = torch.zeros_like(K)
        for b in range(B):
            mm = max(0, min(n, ctx[b] - c0))
            K[b, :mm] = kv[b][0][c0:c0 + mm]
            V[b, :mm] = kv[b][1][c0:c0 + mm]
        bg.blockgtq_quantize_append(cfg, layout, 0, K, V, torch.tensor([c0] * B, dtype=torch.int32, device="cuda"),
                                    cache)
        del K, V
    knew = torch.stack([torch.stack([kv[b][0][ctx[b] + s] for b in range(B)]) for s in range(n_steps)])
    vnew = torch.stack([torch.stack([kv[b][1][ctx[b] + s] for b in range(B)]) for s in range(n_steps)])
    knew = knew[:, None, :, None].contiguous()          # [steps, L, B, 1, H, 128]
    vnew = vnew[:, None, :, None].contiguous()
    q = torch.stack([torch.stack([synth.torch_queries(seed * 16 + b, 0, H * G, [ctx[b] + s], base)[0]
                                  for b in range(B)]) for s in range(n_steps)])[:, None].contiguous()
    base_pos = torch.tensor(ctx, dtype=torch.int32, device="cuda")
    wps = torch.stack([base_pos + s for s in range(n_steps)])
    ctxs = (wps + 1).contiguous()
    max_ctx = Tm
    out = torch.empty((L, B, H * G, 128), dtype=torch.float32, device="cuda")
    ws = torch.zeros(bg.workspace_bytes(cfg, L, 0, max_ctx), dtype=torch.uint8, device="cuda")
    flush = torch.empty(flush_bytes, dtype=torch.uint8, device="cuda")

    def step(s):
        bg.blockgtq_quantize_append(cfg, layout, -1, knew[s], vnew[s], wps[s], cache)
        bg.blockgtq_decode_attn(cfg, layout, -1, q[s], ctxs[s], max_ctx, cache, out=out, workspace=ws)

    for s in range(2):
        step(s)
    st = settle(torch, lambda: step(2), 0.5)
    warm = interleaved(torch, [lambda i: step(4 + i)], args.steps)[0]
    cold_ev = [ev_pair(torch) for _ in range(args.steps)]
    for i in range(args.steps):
        flush.fill_(i & 255)
        cold_ev[i][0].record()
        step(4 + args.steps + i)
        cold_ev[i][1].record()
    torch.cuda.synchronize()
    cold = [a.elapsed_time(b) * 1e3 for a, b in cold_ev]
    ng = n_groups(bits)
    row = (kb * 2 / 8 + 128 * vb / 8 + 2) * H + 2.0 * ng.sum()
    io = B * H * G * 128 * 6
    sb_warm = (sum(ctx) + B * (4 + (args.steps + 1) / 2)) * row + io     # mean context of the warm steps
    sb = (sum(ctx) + B * (4 + args.steps + (args.steps + 1) / 2)) * row + io   # of the cold steps
    fl = np.sum([quantize_flops_per_row(bits[0, h]) for h in range(H)])
    pm = float(np.mean(pre_us))
    res = {"workload": "ragged batch 8, Llama-3.1-8B attention shape (1 layer, 8 KV heads, G = 4), contexts "
                       f"{ctx} (uniform in [4096, 65536]), K3V2, bf16",
           "settle": st, "warm_step_us": stats(warm), "cold_step_us": stats(cold),
           "algorithmic_bytes_per_step": int(sb),
           "warm_gbs": round(sb_warm / (np.median(warm) * 1e-6) / 1e9, 2),
           "cold_gbs": round(sb / (np.median(cold) * 1e-6) / 1e9, 2),
           "cold_pct_hbm_peak": round(100 * sb / (np.median(cold) * 1e-6) / 1e9 / HBM_PEAK_GBS, 2),
           "prefill_16k_call": {"rows": B * chunk * H, "call_us": stats(pre_us),
                                "rows_per_s": round(B * chunk * H / (pm * 1e-6), 1),
                                "roofline": {"bound": "mfma", "achieved": round(B * chunk * fl / (pm * 1e-6) / 1e12, 2),
                                             "peak": FP32_PEAK_TFLOPS, "unit": "TFLOP/s",
                                             "frac": round(B * chunk * fl / (pm * 1e-6) / 1e12 / FP32_PEAK_TFLOPS, 4),
                                             "kernel": "k_quant_rows"}}}
    del cache, layout, flush, knew, vnew, q, out, ws, kv
    torch.cuda.empty_cache()
    return res


def read_probe(bg, torch, nbytes=4 << 30):
    """Plain streaming read of a 4 GiB buffer (library kernel k_read_probe)."""
    src = torch.ones(nbytes, dtype=torch.uint8, device="cuda")
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    for _ in range(3):
        bg.blockgtq_read_probe(src, sink)
    us = interleaved(torch, [lambda i: bg.blockgtq_read_probe(src, sink)], 10)[0]
    del src
    torch.cuda.empty_cache()
    return {"bytes": nbytes, "us": stats(us), "gbs": round(nbytes / (np.median(us) * 1e-6) / 1e9, 1),
            "kernel": "k_read_probe"}


# ------------------------------------------------------------------ CPU oracle baseline

def _cpu_unit_worker(wid, unit, spec, T, bits, budget_s, barrier, queue):
    """One worker process (one BLAS thread): builds the oracle's cache of its
    (layer, KV head) unit from the seeded generators (untimed), waits for the
    other workers, then runs decode steps at positions T, T + 1, ... for
    `budget_s` seconds: encode the appended row, then the rotated-form fp64
    attention of the G query heads over every cached row."""
    try:
        from threadpoolctl import threadpool_limits
        threadpool_limits(1)
    except Exception:  # pragma: no cover
        pass
    from oracle import blockgtq_oracle as o
    from paper_2606_24033_amd import synth
    seed, base, G, vb = spec["seed"], spec["base"], spec["group"], spec["v_bits"]
    layer, h = unit
    extra = 64
    rot_k, rot_v = synth.rotations(seed)
    sig = synth.sigma_profile(seed, layer, h)
    k = synth.cast(synth.keys(seed, layer, h, 0, T + extra, sig, base), "bf16")
    v = synth.cast(synth.values(seed, layer, h, 0, T + extra), "bf16")
    kc, _, kn, _ = o.quantize_keys(k[:T], bits[layer, h], rot_k)
    vc, vn, _ = o.quantize_values(v[:T], rot_v, vb)
    ng = len(np.unique(bits[layer, h]))
    row = spec["k_budget"] * 2 / 8 + 2 * ng + 128 * vb / 8 + 2
    if barrier is not None:
        barrier.wait()
    t0 = time.time()
    nbytes, steps = 0.0, 0
    while steps < extra:
        pos = T + steps
        q = synth.cast(synth.queries(seed, layer, h, pos, G, base, step=steps), "bf16")
        kc1, _, kn1, _ = o.quantize_keys(k[pos:pos + 1], bits[layer, h], rot_k)
        vc1, vn1, _ = o.quantize_values(v[pos:pos + 1], rot_v, vb)
        kc, kn = np.concatenate([kc, kc1]), np.concatenate([kn, kn1])
        vc, vn = np.concatenate([vc, vc1]), np.concatenate([vn, vn1])
        o.attention_rotated(q, kc, kn, bits[layer, h], rot_k, vc, vn, rot_v, vb)
        nbytes += (pos + 1) * row
        steps += 1
        if time.time() - t0 >= budget_s:
            break
    queue.put((wid, t0, time.time(), nbytes, steps))


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def headline_parity(bg, synth, torch, m, units):
    """Parity statistics of the headline workload, part of the CPU-oracle leg
    (the only part of this script that calls the oracle): for a few (layer, KV
    head) units, the fp64 oracle on the same seeded rows (regenerated on the
    device by the same generator call as the prefill, copied to the host)
    against the library's decode of the first step (context T + 1), per query
    head max |out - ref| / max |ref|."""
    from oracle import blockgtq_oracle as o
    G, T = m.G, m.T
    ctx = m.ctxs[0:1].clone()
    out = torch.empty_like(m.out)
    bg.blockgtq_decode_attn(m.cfg, m.layout, -1, m.q[0], ctx, m.max_ctx, m.cache, out=out, workspace=m.ws,
                            n_splits=m.n_splits)
    torch.cuda.synchronize()
    errs = []
    for layer, h in units:
        k, v = synth.torch_layer_kv(m.seed, layer, m.T + m.n_steps, m.sig[layer], m.base)
        kk = k[:T + 1, h].float().cpu().numpy()
        vv = v[:T + 1, h].float().cpu().numpy()
        del k, v
        kc, _, kn, _ = o.quantize_keys(kk, m.bits[layer, h], m.rot_k)
        vc, vn, _ = o.quantize_values(vv, m.rot_v, m.vb)
        q = m.q[0][layer, 0, h * G:(h + 1) * G].float().cpu().numpy()
        ref = o.attention_rotated(q, kc, kn, m.bits[layer, h], m.rot_k, vc, vn, m.rot_v, m.vb)
        got = out[layer, 0, h * G:(h + 1) * G].double().cpu().numpy()
        errs.append(float(np.max(np.abs(got - ref)) / np.max(np.abs(ref))))
    return {"units": [list(u) for u in units], "ctx": T + 1, "max_rel_err": round(max(errs), 7),
            "per_unit": [round(e, 7) for e in errs], "budget": 2e-3,
            "note": "oracle codes from its own fp64 encode; threshold ties (counted in the tests) are not separated"}


def cpu_oracle_baseline(bits, T, workers, spec=LLAMA, budget_s=8.0):
    """The fp64 CPU oracle (rotated form, as it stands) on a bounded sample of
    the headline step: `workers` processes, one host core and one (layer, KV
    head) unit each; after every cache is built, all run decode steps of their
    unit together for `budget_s` seconds.  GB/s of algorithmic bytes over the
    wall time of that phase; the one-thread figure is the mean rate of one
    process in the same phase."""
    import multiprocessing as mp
    ctx = mp.get_context("spawn")
    L, H = spec["n_layers"], spec["n_kv"]
    units = [divmod((w * 37) % (L * H), H) for w in range(workers)]   # spread over layers and heads
    barrier = ctx.Barrier(workers)
    queue = ctx.Queue()
    procs = [ctx.Process(target=_cpu_unit_worker, args=(w, units[w], spec, T, bits, budget_s, barrier, queue))
             for w in range(workers)]
    t_start = time.time()
    for p in procs:
        p.start()
    res = [queue.get(timeout=900) for _ in range(workers)]
    for p in procs:
        p.join(timeout=60)
    t0 = min(r[1] for r in res)
    t1 = max(r[2] for r in res)
    nbytes = sum(r[3] for r in res)
    steps = sum(r[4] for r in res)
    one = float(np.mean([r[3] / (r[2] - r[1]) for r in res]))
    per_step_unit_s = float(np.mean([(r[2] - r[1]) / r[4] for r in res]))
    return {"value": round(nbytes / (t1 - t0) / 1e9, 4), "unit": "GB/s", "cores": int(workers), "kind": "oracle",
            "sample": f"{workers} (layer, KV head) units of the headline step, one process (one thread) each, "
                      f"{steps} decode steps in all at ctx {T + 1}.. (encode the appended row + rotated-form fp64 "
                      f"attention of {spec['group']} query heads), {t1 - t0:.2f} s wall for the timed phase; caches built "
                      f"untimed ({t0 - t_start:.1f} s)",
            "one_thread_gbs": round(one / 1e9, 4), "one_thread_s_per_unit_step": round(per_step_unit_s, 3),
            "cpu_model": _cpu_model(), "host_cpus": len(os.sched_getaffinity(0)),
            "us_per_step_equiv": round(per_step_unit_s * L * H / workers * 1e6, 1)}


# ------------------------------------------------------------------ main

def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for {args.gpus}); multi-GPU runs are not part of this build.",
              file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2606_24033_amd import blockgtq as bg
    from paper_2606_24033_amd import synth

    if not torch.cuda.is_available():
        print("no GPU available", file=sys.stderr)
        sys.exit(1)
    bg.lib()
    T = args.ctx
    W, K = args.warmup, args.steps
    want_fp16 = not args.no_fp16 and not args.only_headline
    want_win = not args.no_protected and not args.only_headline
    t_setup = time.time()
    spec = LLAMA if args.model == "llama8b_k2v2" else QWEN_LONG
    m = Model(bg, synth, torch, spec, T, W + K, fp16=want_fp16, window=want_win, n_splits=args.n_splits,
              chunk=None if spec is LLAMA else 8192)
    log(f"setup {time.time() - t_setup:.1f} s (prefill of {T} rows x {m.L} layers x {m.H} heads)")
    if args.copy_calib_mib > 0:
        # a plain copy of known size: FETCH_SIZE / WRITE_SIZE of this dispatch
        # calibrate the same counters taken on the decode kernel
        n = args.copy_calib_mib << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"calibration copy: {n} bytes read, {n} bytes written")
        del src, dst

    for s in range(W):
        m.step(s)
    torch.cuda.synchronize()
    settled = settle(torch, lambda: m.step(W), args.settle_s)
    t_wall = time.perf_counter()
    step_us, dec_us, total_ms = timed_steps(torch, m, W, K)
    wall = time.perf_counter() - t_wall
    ms_per_step = total_ms / K
    log(f"settle {settled}; timed {K} steps: {total_ms:.2f} ms on events, {wall * 1e3:.2f} ms wall")

    ctx_mean = T + W + (K + 1) / 2.0
    step_bytes = m.step_bytes(ctx_mean)
    gbs = step_bytes / (ms_per_step * 1e-3) / 1e9
    dec_mean = float(np.mean(dec_us))
    dec_gbs = step_bytes / (dec_mean * 1e-6) / 1e9

    result = {
        "metric": "packed-KV decode attention µs/step + effective HBM GB/s (% of peak) at 128K ctx",
        "value": round(gbs, 2), "unit": "GB/s", "n_gpus": 1, "steps": K, "warmup": W,
        "ms_per_step": round(ms_per_step, 4), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f16", "data": "synthetic",
        "config": {"workload": ("Llama-3.1-8B-shaped full decode step: 32 layers x 8 KV heads (32 q heads), "
                                f"d_h 128, {T} cached rows, K2V2, batch 1, bf16 inputs") if spec is LLAMA else
                               ("Qwen2.5-3B-shaped full decode step: 36 layers x 2 KV heads (16 q heads), "
                                f"d_h 128, {T} cached rows, K3V3, batch 1, bf16 inputs"),
                   "global_batch": 1, "seq_len": T, "parallelism": "none (1 GPU)", "n_splits": args.n_splits},
        "settle": settled,
        "us_per_step": round(ms_per_step * 1e3, 2),
        "us_per_step_median": round(float(np.median(step_us)), 2),
        "us_per_step_p5": round(float(np.percentile(step_us, 5)), 2),
        "us_per_step_p95": round(float(np.percentile(step_us, 95)), 2),
        "pct_hbm_peak": round(100 * gbs / HBM_PEAK_GBS, 2),
        "decode_call_us_mean": round(dec_mean, 2),
        "decode_call_us_median": round(float(np.median(dec_us)), 2),
        "packed_bytes_per_step": int(step_bytes),
        "fp16_bytes_per_step": int(m.fp16_bytes(ctx_mean)),
    }
    traffic = measured_traffic()
    result["roofline"] = {"bound": "hbm", "achieved": round(dec_gbs, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                          "frac": round(dec_gbs / HBM_PEAK_GBS, 4),
                          "traffic": None if traffic is None else int(traffic),
                          "kernel": "k_split_mfma (one launch per decode call: query rotation, split pass, "
                                    f"merge), all {m.L} layers",
                          "algorithmic_bytes_per_launch": int(step_bytes),
                          "launch_us_mean": round(dec_mean, 2),
                          "launch_us_median": round(float(np.median(dec_us)), 2)}
    if not args.only_headline:
        rp = read_probe(bg, torch)
        result["read_probe"] = rp
        result["roofline"]["read_probe_gbs"] = rp["gbs"]
        result["roofline"]["frac_of_read_probe"] = round(dec_gbs / rp["gbs"], 4)
        result["quantize_prefill"] = quantize_roofline(
            m, f"prefill quantize_append of {T} rows x 8 KV heads per call (one call per layer), Llama-3.1-8B "
               "shape, K2V2, bf16")

    parity = None
    if not args.no_cpu and not args.only_headline:
        parity = headline_parity(bg, synth, torch, m, [(5, 3), (27, 6)])
        log(f"headline parity {parity['max_rel_err']}")
    if want_fp16:
        out16 = torch.empty_like(m.out)
        p_us, f_us = interleaved(torch, [lambda i: m.decode(W + i), lambda i: m.decode_fp16(W + i, out16)], K)
        fbytes = m.fp16_bytes(ctx_mean) + m.io_bytes()
        result["fp16_decode_us_median"] = round(float(np.median(f_us)), 2)
        result["fp16_decode_gbs"] = round(fbytes / (np.mean(f_us) * 1e-6) / 1e9, 2)
        result["fp16_decode_pct_hbm_peak"] = round(100 * fbytes / (np.mean(f_us) * 1e-6) / 1e9 / HBM_PEAK_GBS, 2)
        result["packed_decode_us_median_interleaved"] = round(float(np.median(p_us)), 2)
        result["speedup_vs_fp16_decode"] = round(float(np.median(f_us) / np.median(p_us)), 3)
        sd = sdpa_decode_context(torch, m, W, K)
        if sd is not None:
            result["torch_sdpa_fp16_decode"] = sd
        del m.k16, m.v16
        torch.cuda.empty_cache()

    if want_win:
        result["protected_window"] = protected_measurement(bg, torch, m, args, W)
        del m.window

    if not args.no_uniform and not args.only_headline:
        result["uniform_tq_mse"] = uniform_comparison(bg, synth, torch, m, args, W)

    if not args.no_rope_step and not args.only_headline:
        result["rope_step"] = rope_step_measurement(bg, torch, m, args, W)
        result["per_layer_graph"] = per_layer_graph_measurement(bg, torch, m, args, W)

    if not args.no_prefill and not args.only_headline:
        result["prefill_attn"] = prefill_measurement(bg, synth, torch, m, args.prefill_len)
    bits_llama = m.bits.copy()
    m.free()
    del m

    if not args.no_workloads and not args.only_headline:
        wl = {}
        toy = Model(bg, synth, torch, dict(name="toy", seed=1, n_layers=1, n_kv=1, group=4, base=1e4, k_budget=192,
                                           v_bits=2), 2048, W + K, in_dtype=bg.BGTQ_FP32, n_cal=256)
        wl["toy_single_head"] = workload_line(torch, toy, args, "toy single head: 1 layer, 1 KV head, G = 4, "
                                              "base 1e4, 2048 fp32 rows, K3V2 (latency-bound; report us only)", 0.3,
                                              cold=True)
        toy.free()
        q2 = Model(bg, synth, torch, dict(name="Qwen2.5-3B", seed=2, n_layers=1, n_kv=2, group=8, base=1e6,
                                          k_budget=192, v_bits=3), 32768, max(64, W + K))
        K64 = argparse.Namespace(**{**vars(args), "steps": 64, "warmup": 0})
        line = workload_line(torch, q2, K64, "Qwen2.5-3B-shaped layer: 16 q / 2 KV heads, base 1e6, bf16, "
                             "32768 rows, K3V3; 64 decode steps", 0.3, cold=True)
        wp0 = torch.zeros(1, dtype=torch.int32, device="cuda")
        kk, vv = synth.torch_layer_kv(2, 0, 32768, q2.sig[0], q2.base)
        kk, vv = kk[None].contiguous(), vv[None].contiguous()
        for _ in range(2):
            bg.blockgtq_quantize_append(q2.cfg, q2.layout, 0, kk, vv, wp0, q2.cache)
        pre = interleaved(torch, [lambda i: bg.blockgtq_quantize_append(q2.cfg, q2.layout, 0, kk, vv, wp0, q2.cache)],
                          5)[0]
        line["prefill_call_us"] = stats(pre)
        line["prefill_rows_per_s"] = round(32768 * 2 / (np.median(pre) * 1e-6), 1)
        del kk, vv
        wl["qwen3b_layer_32k"] = line
        q2.free()
        for Tq in ([131072] if args.no_long else [131072, 262144, 524288]):
            mq = Model(bg, synth, torch, QWEN_LONG, Tq, W + K, chunk=8192, fp16=want_fp16, n_splits=args.n_splits)
            lab = (f"Qwen2.5-3B-shaped decode step: 36 layers x 2 KV heads (16 q heads, G = 8), base 1e6, bf16, "
                   f"{Tq} rows prefilled in 8192-row chunks, K3V3")
            wl[f"qwen3b_k3v3_{Tq // 1024}k"] = workload_line(torch, mq, args, lab, 0.5, fp16=want_fp16)
            if Tq == 131072:
                result["quantize_prefill_qwen_8k_chunks"] = quantize_roofline(
                    mq, "prefill quantize_append of 8192-row chunks x 2 KV heads, Qwen2.5-3B shape, K3V3, bf16")
            mq.free()
            del mq
            log(f"workload qwen {Tq} done")
        wl["ragged_batch8"] = ragged_workload(bg, synth, torch, args)
        result["workloads"] = wl

    if not args.no_cpu and not args.only_headline:
        workers = args.cpu_workers or min(16, len(os.sched_getaffinity(0)))
        result["cpu_baseline"] = cpu_oracle_baseline(bits_llama, T, workers, spec)
        if parity is not None:
            result["cpu_baseline"]["headline_parity"] = parity
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
