#!/usr/bin/env python3
"""Benchmark: one rank's qwZ / qgZ compression step for a GPT-20B layer on one MI355X.

A step is one pass of the whole path over one GPT-20B-shaped layer
(hidden 6144, FFN 24576: 452,984,832 parameters), inputs resident in HBM:

  qwz_quantize      bf16 weight shard (1/8 = 56,623,104), INT8 blocks of 256,
                    written into its slot of the gathered buffer
  qwz_dequantize    the gathered INT8 layer (452,984,832) -> bf16
  qgz_quantize      fp32 gradient of the layer (452,984,832), INT4 blocks of 128
  qgz_reduce_level  P = 8 slices of 56,623,104 (one intra-node level)
  qgz_dequantize    the reduced 56,623,104-element shard -> fp32
  qgz_reduce_level  3-level chain: P = 2 (m 226,492,416), P = 4 (m 56,623,104),
                    P = 48 (m 1,179,648)
  qgz_dequantize    the final 1,179,648-element shard -> fp32

The collectives between the calls (the weight Allgather, the gradient
all-to-all of each level) are outside this path: their results are placed
in HBM before timing (peer slices are quantised from seeded fp32 peer
gradients; a level's local slice is chunk 0 of the previous level's output).

Timing of the step: W warm-up steps; a breakdown pass of K steps with HIP
events between all calls (the per-call event figures); then --settle more
steps, because the GPU's clock drops for some tens of milliseconds once
continuous heavy work starts (measured: 2.15 -> 1.57 -> 2.2 GHz over ~60
launches of the reduce level, and the step from 0.84 to a steady 0.75 ms
over its first ~40 steps; the breakdown pass's events leave idle gaps that
let the clock rise again); then the timed region of K steps, host wall clock
between two device synchronisations, with one event pair around the
dominant kernel in every fourth step only (--dom-every; its per-launch
duration gives the roofline figure).
All events are HIP events without the system-scope fence (TimingEvent):
torch's default events write back and invalidate the caches when recorded
and cost about 3 us of GPU time each, fence-free ones about 1.7 us.
The settle steps' times are reported too.

Per-call figures (`kernels`): each call of the step launched back to back in
a loop, its inputs rotating over copies totalling >= 1 GB so the 256 MB
last-level cache cannot serve them (loop time / launches, which includes
the GPU's gap between dependent launches); beside it the call's time inside
the step's breakdown pass (event brackets), and the kernel-only duration
from the committed rocprofv3 trace when that was taken on these sources.

Output: one JSON line.  value = algorithmic bytes of the step / step time.
Extra fields, measured after the timed region: the other workloads
(tiny-1024x1024, gpt-1.3b-layer, outlier-edge-123456789) call by call; the
bandwidth ceilings of hand-written copy / read / write / P-stream kernels
(libzq_probe.so); the last level fused with the final dequantisation, the
degree-2 weight shard, the P = 8 level in all-shares mode (m = n) and
reading its slices in place from separate buffers, and the layer's forward
GEMMs with the INT8 weight dequantised on load against dequantise + torch's
GEMM.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "achieved HBM GB/s (% of MI355X peak) for qwZ quant/dequant + qgZ reduce, GPT-20B layer"
HBM_PEAK_GBPS = 8000.0
WBLOCK, GBLOCK, SHARD = 256, 128, 8
FANINS = [2, 4, 48]


def nsc(n, b):
    return (n + b - 1) // b


def nb4(n):
    return (n + 1) // 2


# algorithmic bytes per call (what the method must read and write)
def bytes_qwz_quant(n, in_b, block):
    return n * in_b + n + 4 * nsc(n, block)


def bytes_qwz_deq(n, out_b, block):
    return n + 4 * nsc(n, block) + n * out_b


def bytes_qgz_quant(n, in_b, block):
    return n * in_b + nb4(n) + 4 * nsc(n, block)


def bytes_reduce(P, m, block):
    return (P + 1) * (nb4(m) + 4 * nsc(m, block))


def bytes_qgz_deq(n, out_b, block):
    return nb4(n) + 4 * nsc(n, block) + n * out_b


class Layer20B:
    """Device buffers and the launch sequence of one step."""

    def __init__(self, n, log):
        import numpy as np
        import torch

        import paper_2501_04266_amd as zq
        from paper_2501_04266_amd import workloads as wl

        self.zq, self.torch, self.np = zq, torch, np
        self.n = n
        dev = "cuda"
        T = torch
        t0 = time.time()
        self.host = {}
        # weights: bf16 N(0, 0.02); the gathered INT8 layer is the Allgather of
        # all 8 shards' codes, which (shards being block-aligned) equals the
        # quantisation of the whole layer
        w = wl.weights(n, "bf16", key=[3, wl.ROLE_WEIGHT, 0, 0])
        self.host["w"] = w
        self.w = T.from_numpy(w.view(np.int16)).to(dev).view(T.bfloat16)
        self.shard = n // SHARD
        self.codes = T.empty(n, dtype=T.int8, device=dev)
        self.wscales = T.empty(nsc(n, WBLOCK), dtype=T.float32, device=dev)
        zq.qwz_quantize(self.w, WBLOCK, codes=self.codes, scales=self.wscales)
        self.y = T.empty(n, dtype=T.bfloat16, device=dev)
        log(f"weights ready ({time.time() - t0:.1f}s)")

        # own fp32 gradient N(0, 1e-3) and its INT4 wire format
        g = wl.normal_f32(n, 1e-3, key=[3, wl.ROLE_OWN_GRAD, 0, 0])
        self.host["g"] = g
        self.g = T.from_numpy(g).to(dev)
        self.gp = T.empty(nb4(n), dtype=T.uint8, device=dev)
        self.gs = T.empty(nsc(n, GBLOCK), dtype=T.float32, device=dev)
        zq.qgz_quantize(self.g, GBLOCK, packed=self.gp, scales=self.gs)
        log(f"gradient ready ({time.time() - t0:.1f}s)")

        # one intra-node level, P = 8 (local rank 0)
        self.m8 = n // 8
        self.d8 = self._level_buffers(8, self.m8, self.gp, self.gs, key=(3, 0))
        self.o8 = (T.empty(nb4(self.m8), dtype=T.uint8, device=dev), T.empty(nsc(self.m8, GBLOCK), device=dev))
        self.gshard = T.empty(self.m8, dtype=T.float32, device=dev)
        log(f"P=8 level ready ({time.time() - t0:.1f}s)")

        # 3-level chain 2 / 4 / 48
        self.chain = []
        cur_p, cur_s, cur_m = self.gp, self.gs, n
        for k, P in enumerate(FANINS):
            m = cur_m // P
            d = self._level_buffers(P, m, cur_p, cur_s, key=(4, k))
            o = (T.empty(nb4(m), dtype=T.uint8, device=dev), T.empty(nsc(m, GBLOCK), device=dev))
            zq.qgz_reduce_level(d[0], d[1], P, m, GBLOCK, packed_out=o[0], scales_out=o[1])
            self.chain.append((P, m, d, o))
            cur_p, cur_s, cur_m = o[0], o[1], m
        self.final = T.empty(cur_m, dtype=T.float32, device=dev)
        T.cuda.synchronize()
        log(f"3-level chain ready ({time.time() - t0:.1f}s)")

        # (name, algorithmic bytes, elements) of each launch, in step order;
        # elements = the elements of the tensor a call codes (P*m slice
        # elements for a reduce level)
        self.calls = [
            ("qwz_quantize", bytes_qwz_quant(self.shard, 2, WBLOCK), self.shard),
            ("qwz_dequantize", bytes_qwz_deq(n, 2, WBLOCK), n),
            ("qgz_quantize", bytes_qgz_quant(n, 4, GBLOCK), n),
            ("qgz_reduce_level P=8", bytes_reduce(8, self.m8, GBLOCK), 8 * self.m8),
            ("qgz_dequantize P=8 shard", bytes_qgz_deq(self.m8, 4, GBLOCK), self.m8),
        ] + [(f"qgz_reduce_level P={P}", bytes_reduce(P, m, GBLOCK), P * m) for P, m, _, _ in self.chain] + [
            ("qgz_dequantize chain shard", bytes_qgz_deq(cur_m, 4, GBLOCK), cur_m)]

    def _level_buffers(self, P, m, own_p, own_s, key):
        """All-to-all receive buffer of one level at local rank 0: slice 0 is
        chunk 0 of the local input, slices 1..P-1 are INT4 quantisations of
        seeded fp32 peer chunks."""
        np, T, zq = self.np, self.torch, self.zq
        from paper_2501_04266_amd import workloads as wl
        mb, ms = nb4(m), nsc(m, GBLOCK)
        pin = T.empty(P * mb, dtype=T.uint8, device="cuda")
        sin = T.empty(P * ms, dtype=T.float32, device="cuda")
        pin[:mb].copy_(own_p[:mb])
        sin[:ms].copy_(own_s[:ms])
        peers = []
        for p in range(1, P):
            xs = wl.normal_f32(m, 1e-3, key=[key[0], wl.ROLE_PEER_GRAD, key[1], p])
            peers.append(xs)
            zq.qgz_quantize(T.from_numpy(xs).to("cuda"), GBLOCK, packed=pin[p * mb:(p + 1) * mb],
                            scales=sin[p * ms:(p + 1) * ms])
        self.host[("peers",) + tuple(key)] = peers
        return pin, sin

    def step(self, ev=None, around=None):
        """One pass of the path.  ev: events recorded before the first call,
        between calls and after the last (len(calls) + 1 of them); with
        `around` = i, only the pair ev[0], ev[1] around call i."""
        zq = self.zq
        n, s = self.n, self.shard

        def mark(i):
            if ev is None:
                return
            if around is None:
                ev[i].record()
            elif i == around:
                ev[0].record()
            elif i == around + 1:
                ev[1].record()

        mark(0)
        zq.qwz_quantize(self.w[:s], WBLOCK, codes=self.codes[:s], scales=self.wscales[:nsc(s, WBLOCK)])
        mark(1)
        zq.qwz_dequantize(self.codes, self.wscales, WBLOCK, y=self.y)
        mark(2)
        zq.qgz_quantize(self.g, GBLOCK, packed=self.gp, scales=self.gs)
        mark(3)
        zq.qgz_reduce_level(self.d8[0], self.d8[1], 8, self.m8, GBLOCK, packed_out=self.o8[0], scales_out=self.o8[1])
        mark(4)
        zq.qgz_dequantize(self.o8[0], self.o8[1], self.m8, GBLOCK, y=self.gshard)
        mark(5)
        i = 5
        for P, m, d, o in self.chain:
            zq.qgz_reduce_level(d[0], d[1], P, m, GBLOCK, packed_out=o[0], scales_out=o[1])
            i += 1
            mark(i)
        P, m, d, o = self.chain[-1]
        zq.qgz_dequantize(o[0], o[1], m, GBLOCK, y=self.final)
        mark(i + 1)


def oracle_step(L, threads, repeats=1):
    """The same step on the CPU oracle over the same host inputs; returns
    (mean seconds per step in the timed calls, outputs).  Each timed call runs
    `repeats` times.  Preparation (gathered codes, peer slices) is untimed, as
    on the GPU."""
    import numpy as np

    import oracle
    oracle.set_threads(threads)
    n, s = L.n, L.shard
    w, g = L.host["w"], L.host["g"]
    codes_all, sc_all = oracle.qwz_quantize(w, WBLOCK, "bf16")       # the gathered layer (prep)
    outs, t = {}, 0.0
    per_call = []

    def timed(fn, *a):
        nonlocal t
        t0 = time.perf_counter()
        for _ in range(repeats):
            r = fn(*a)
        dt = (time.perf_counter() - t0) / repeats
        t += dt
        per_call.append(round(dt, 4))
        return r

    outs["shard_codes"] = timed(oracle.qwz_quantize, w[:s], WBLOCK, "bf16")
    outs["y"] = timed(oracle.qwz_dequantize, codes_all, sc_all, WBLOCK, "bf16")
    gp, gs = timed(oracle.qgz_quantize, g, GBLOCK, "f32")

    def level(P, m, own_p, own_s, key):
        mb, ms = nb4(m), nsc(m, GBLOCK)
        ps, ss = [own_p[:mb]], [own_s[:ms]]
        for xs in L.host[("peers",) + key]:
            a, b = oracle.qgz_quantize(xs, GBLOCK, "f32")
            ps.append(a)
            ss.append(b)
        return np.concatenate(ps), np.concatenate(ss)

    pin, sin = level(8, L.m8, gp, gs, (3, 0))
    o8 = timed(oracle.qgz_reduce_level, pin, sin, 8, L.m8, GBLOCK)
    outs["gshard"] = timed(oracle.qgz_dequantize, o8[0], o8[1], L.m8, GBLOCK, "f32")
    cur_p, cur_s, cur_m = gp, gs, n
    for k, P in enumerate(FANINS):
        m = cur_m // P
        pin, sin = level(P, m, cur_p, cur_s, (4, k))
        cur_p, cur_s = timed(oracle.qgz_reduce_level, pin, sin, P, m, GBLOCK)
        outs[f"chain{k}"] = (cur_p, cur_s)
        cur_m = m
    outs["final"] = timed(oracle.qgz_dequantize, cur_p, cur_s, cur_m, GBLOCK, "f32")
    outs["gp"] = (gp, gs)
    outs["per_call_s"] = per_call
    return t, outs


def check_against_oracle(L, outs):
    """Bit-exact comparison of every step output with the oracle's."""
    import numpy as np
    T = L.torch

    def host(t):
        if t.dtype == T.bfloat16:
            return t.view(T.int16).cpu().numpy().view(np.uint16)
        return t.cpu().numpy()

    pairs = [
        ("shard codes", host(L.codes[:L.shard]), outs["shard_codes"][0]),
        ("shard scales", host(L.wscales[:nsc(L.shard, WBLOCK)]), outs["shard_codes"][1]),
        ("dequant bf16", host(L.y), outs["y"]),
        ("grad packed", host(L.gp), outs["gp"][0]),
        ("grad scales", host(L.gs), outs["gp"][1]),
        ("P=8 shard fp32", host(L.gshard), outs["gshard"]),
        ("final fp32", host(L.final), outs["final"]),
    ]
    for k, (P, m, d, o) in enumerate(L.chain):
        pairs.append((f"chain level {k} packed", host(o[0]), outs[f"chain{k}"][0]))
        pairs.append((f"chain level {k} scales", host(o[1]), outs[f"chain{k}"][1]))
    bad = [name for name, a, b in pairs if a.tobytes() != np.ascontiguousarray(b).tobytes()]
    return bad


KERNEL_SOURCES = [os.path.join(ROOT, "paper_2501_04266_amd", "csrc", f)
                  for f in ("zq_kernels.hip", "zq_internal.h", "zq_device.h", "zq_host.h", "zq_api.hip")]
TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "gpt20b_step_pmc_traffic.txt")
VALU_PROFILE = os.path.join(ROOT, "profiles", "gpt20b_step_pmc_valu.txt")


def kernel_source_hash():
    import hashlib
    return hashlib.sha256(b"".join(open(p, "rb").read() for p in KERNEL_SOURCES)).hexdigest()[:16]


def load_traffic(call):
    """HBM bytes per launch of `call` from the committed rocprofv3 PMC summary
    (FETCH_SIZE and WRITE_SIZE runs, calibrated on a plain copy), or None when
    there is none or it was taken on different kernel sources."""
    if not os.path.exists(TRAFFIC_PROFILE):
        return None
    lines = open(TRAFFIC_PROFILE).read().splitlines()
    tag = "# kernel source sha256[:16]:"
    h = next((ln[len(tag):].strip() for ln in lines if ln.startswith(tag)), None)
    if h != kernel_source_hash():
        return None
    for ln in lines:
        if ln.startswith(call + " ") and not ln.startswith("#"):
            rest = ln[len(call):].split()
            return int(rest[2])
    return None


def load_valu(call):
    """VALU figures per launch of `call` from the committed rocprofv3 PMC summary
    (SQ_INSTS_VALU, GRBM_GUI_ACTIVE), or None when there is none for the call or
    it was taken on different kernel sources."""
    if not os.path.exists(VALU_PROFILE):
        return None
    lines = open(VALU_PROFILE).read().splitlines()
    tag = "# kernel source sha256[:16]:"
    h = next((ln[len(tag):].strip() for ln in lines if ln.startswith(tag)), None)
    if h != kernel_source_hash():
        return None
    for ln in lines:
        if ln.startswith(call + " ") and not ln.startswith("#"):
            rest = ln[len(call):].split()
            return {"valu_insts_per_elem": float(rest[1]), "valu_busy": float(rest[3])}
    return None


GEMM_TOKENS = 8192
SMALL_TOKENS = 64
DECODE_TOKENS = 16
MFMA_BF16_PEAK_TFLOPS = 2500.0


def gemm_figures(L, reps, log):
    """The GPT-20B layer's four forward GEMMs (QKV 3h x h, attention out h x h,
    FC1 4h x h, FC2 h x 4h) over GEMM_TOKENS rows of bf16 activations, weights
    from the gathered INT8 layer: fused dequantise-on-load vs qwz_dequantize of
    the layer followed by torch's bf16 GEMM (hipBLASLt)."""
    import torch
    import torch.nn.functional as F
    zq = L.zq
    h, M, B = 6144, GEMM_TOKENS, WBLOCK
    shapes = (("qkv", 3 * h, h), ("attn_out", h, h), ("fc1", 4 * h, h), ("fc2", h, 4 * h))
    g = torch.Generator(device="cuda")
    g.manual_seed(20250104)
    xs = {K: torch.randn((M, K), device="cuda", dtype=torch.bfloat16, generator=g) for K in (h, 4 * h)}
    ys = {name: torch.empty((M, N), device="cuda", dtype=torch.float32) for name, N, _ in shapes}
    slices = []
    off = 0
    for name, N, K in shapes:
        slices.append((name, N, K, L.codes[off:off + N * K], L.wscales[off // B:(off + N * K) // B]))
        off += N * K

    def fused():
        for name, N, K, c, sc in slices:
            zq.qwz_dequant_gemm(xs[K], c, sc, N, B, y=ys[name])

    def separate():
        zq.qwz_dequantize(L.codes, L.wscales, B, y=L.y)
        o = 0
        for name, N, K, _, _ in slices:
            F.linear(xs[K], L.y[o:o + N * K].view(N, K))
            o += N * K

    def timed(fn):
        for _ in range(2):
            fn()
        e0, e1 = TimingEvent(), TimingEvent()
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    # the same GEMMs over few rows, where the weight stream dominates: fused
    # vs separate, at SMALL_TOKENS (the ping-pong kernel's 128-row tiles) and
    # DECODE_TOKENS (the weight-streaming kernel)
    wbytes = L.codes.numel() + 4 * L.wscales.numel()

    def few_rows(T):
        xs_small = {K: xs[K][:T] for K in (h, 4 * h)}
        ys_small = {name: torch.empty((T, N), device="cuda", dtype=torch.float32) for name, N, _ in shapes}

        def fused_small():
            for name, N, K, c, sc in slices:
                zq.qwz_dequant_gemm(xs_small[K], c, sc, N, B, y=ys_small[name])

        def separate_small():
            zq.qwz_dequantize(L.codes, L.wscales, B, y=L.y)
            o = 0
            for name, N, K, _, _ in slices:
                F.linear(xs_small[K], L.y[o:o + N * K].view(N, K))
                o += N * K

        r = {"tokens": T, "fused_ms": round(timed(fused_small), 4), "separate_ms": round(timed(separate_small), 4)}
        r["fused_weight_GBps"] = round(wbytes / (r["fused_ms"] * 1e-3) / 1e9, 1)
        return r

    small, decode = few_rows(SMALL_TOKENS), few_rows(DECODE_TOKENS)

    flops = sum(2 * M * N * K for _, N, K in shapes)
    f_ms, s_ms = timed(fused), timed(separate)
    per = {}
    for name, N, K, c, sc in slices:
        ms = timed(lambda: zq.qwz_dequant_gemm(xs[K], c, sc, N, B, y=ys[name]))
        per[name] = round(2 * M * N * K / (ms * 1e-3) / 1e12, 1)
    tf = flops / (f_ms * 1e-3) / 1e12
    log(f"dequant GEMM: fused {f_ms:.3f} ms ({tf:.0f} TFLOP/s), separate {s_ms:.3f} ms")
    return {"tokens": M, "flops": flops, "fused_ms": round(f_ms, 3), "fused_TFLOPs": round(tf, 1),
            "roofline": {"bound": "mfma", "achieved": round(tf, 1), "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                         "frac": round(tf / MFMA_BF16_PEAK_TFLOPS, 4)},
            "per_gemm_TFLOPs": per,
            "separate_dequant_plus_torch_gemm_ms": round(s_ms, 3),
            "separate_TFLOPs": round(flops / (s_ms * 1e-3) / 1e12, 1),
            "few_tokens": small, "decode_tokens": decode}


def cpu_model():
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


ROT_BYTES = 1100 * 1000 * 1000   # inputs + outputs rotated per call loop: beyond the 256 MB last-level cache
GATE_BYTES = 100 * 1000 * 1000   # calls of at least this many bytes are held to 70% of HBM peak
ALL_SHARES_SETTLE_S = 0.1
TRACE_PROFILE = os.path.join(ROOT, "profiles", "gpt20b_step_kernel_trace.txt")


def _tensor_bytes(ts):
    return sum(t.numel() * t.element_size() for t in ts)


HIP_EVENT_DISABLE_SYSTEM_FENCE = 0x20000000  # hipEventDisableSystemFence


class TimingEvent:
    """A HIP event used only to take GPU timestamps, recorded on torch's
    current stream (where the bindings launch).

    It is created with hipEventDisableSystemFence: recording it does not
    write back and invalidate the caches at system scope, which a default
    event (torch.cuda.Event) does and which leaves a gap of several
    microseconds between the launches around it.  Read it (elapsed_time)
    only after a device synchronisation."""

    _hip = None

    @classmethod
    def _runtime(cls):
        if cls._hip is None:
            import ctypes

            import torch  # noqa: F401  (loads the HIP runtime that torch's streams belong to)
            path = next((ln.split()[-1] for ln in open("/proc/self/maps") if "libamdhip64.so" in ln),
                        "libamdhip64.so")
            hip = ctypes.CDLL(path)
            vp = ctypes.c_void_p
            hip.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(vp), ctypes.c_uint]
            hip.hipEventRecord.argtypes = [vp, vp]
            hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), vp, vp]
            hip.hipEventDestroy.argtypes = [vp]
            for f in (hip.hipEventCreateWithFlags, hip.hipEventRecord, hip.hipEventElapsedTime,
                      hip.hipEventDestroy):
                f.restype = ctypes.c_int
            cls._hip = hip
        return cls._hip

    def __init__(self):
        import ctypes
        self._hip = self._runtime()
        self.h = ctypes.c_void_p()
        self._check(self._hip.hipEventCreateWithFlags(ctypes.byref(self.h), HIP_EVENT_DISABLE_SYSTEM_FENCE),
                    "hipEventCreateWithFlags")

    @staticmethod
    def _check(rc, what):
        if rc != 0:
            raise RuntimeError(f"{what} failed with HIP error {rc}")

    def record(self):
        import torch
        self._check(self._hip.hipEventRecord(self.h, torch.cuda.current_stream().cuda_stream), "hipEventRecord")

    def elapsed_time(self, end):
        """Milliseconds from this event to `end`."""
        import ctypes
        ms = ctypes.c_float()
        self._check(self._hip.hipEventElapsedTime(ctypes.byref(ms), self.h, end.h), "hipEventElapsedTime")
        return ms.value

    def __del__(self):
        # not at interpreter exit: the runtime may already be torn down then
        h = getattr(self, "h", None)
        if h is not None and h.value and not sys.is_finalizing():
            self._hip.hipEventDestroy(h)


def rotation_runs(fn, inputs, outputs, footprint=None):
    """Closures running fn(inputs, outputs) over enough copies of the inputs
    (and separate outputs) that one pass over them moves >= ROT_BYTES: a loop
    over them streams from HBM, not from the last-level cache.  Copy 0 is the
    given buffers."""
    import torch
    fp = footprint or _tensor_bytes(inputs) + _tensor_bytes(outputs)
    nsets = max(1, -(-ROT_BYTES // max(1, fp)))
    runs = [lambda: fn(inputs, outputs)]
    for _ in range(1, nsets):
        ins = [t.clone() for t in inputs]
        outs = [torch.empty_like(t) for t in outputs]
        runs.append(lambda ins=ins, outs=outs: fn(ins, outs))
    return runs


def loop_us(runs, reps, warm=3):
    """Mean microseconds per launch over `reps` back-to-back launches cycling
    through `runs` (events around the whole loop only)."""
    import torch
    for i in range(warm):
        runs[i % len(runs)]()
    e0, e1 = TimingEvent(), TimingEvent()
    e0.record()
    for i in range(reps):
        runs[i % len(runs)]()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1e3 / reps


def call_figures(name, nbytes, elems, us, nsets=None):
    r = {"call": name, "bytes": nbytes, "elements": elems, "us": round(us, 2),
         "GBps": round(nbytes / (us * 1e-6) / 1e9, 1), "Gelem_per_s": round(elems / (us * 1e-6) / 1e9, 1),
         "pct_hbm_peak": round(100 * nbytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBPS, 1)}
    if nsets is not None:
        r["rotated_sets"] = nsets
    return r


def timed_calls(specs, reps):
    """specs: (name, bytes, elements, fn, inputs, outputs) -> per-call figures
    from rotated back-to-back loops."""
    import torch
    out = []
    for name, nbytes, elems, fn, ins, outs in specs:
        runs = rotation_runs(fn, ins, outs)
        us = loop_us(runs, max(reps, 2 * len(runs)))
        out.append(call_figures(name, nbytes, elems, us, len(runs)))
        del runs
        torch.cuda.empty_cache()
    return out


def load_trace(call):
    """Kernel-only microseconds per launch of `call` in the step, from the
    committed rocprofv3 kernel trace, or None when there is none or it was
    taken on different kernel sources."""
    if not os.path.exists(TRACE_PROFILE):
        return None
    lines = open(TRACE_PROFILE).read().splitlines()
    tag = "# kernel source sha256[:16]:"
    h = next((ln[len(tag):].strip() for ln in lines if ln.startswith(tag)), None)
    if h != kernel_source_hash():
        return None
    for ln in lines:
        if ln.startswith(call + "  ") and not ln.startswith("#"):
            rest = ln[len(call):].split()
            return float(rest[-4])
    return None


class Probe:
    """The bandwidth-ceiling kernels of libzq_probe.so (copy, read, write,
    P read streams + one write stream, 8 bytes in + 16 out per thread)."""

    def __init__(self):
        import ctypes

        import torch
        from paper_2501_04266_amd import build as zbuild
        if not os.path.exists(zbuild.PROBE_LIB):
            raise ImportError(f"{zbuild.PROBE_LIB} is not built; run `python -m paper_2501_04266_amd.build`")
        L = ctypes.CDLL(zbuild.PROBE_LIB)
        vp, i64, i32, u32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_uint32
        for name, args in {"zqp_copy": [vp, vp, i64, vp], "zqp_read": [vp, i64, vp, u32, vp],
                           "zqp_write": [vp, i64, u32, vp], "zqp_streams": [vp, i32, i64, vp, vp],
                           "zqp_expand": [vp, i64, vp, vp]}.items():
            getattr(L, name).argtypes, getattr(L, name).restype = args, ctypes.c_int
        self.L, self.torch = L, torch

    def _st(self):
        return self.torch.cuda.current_stream().cuda_stream

    def _ok(self, rc, what):
        if rc != 0:
            raise RuntimeError(f"{what} failed ({rc})")

    def ceilings(self, reps=20):
        """GB/s of each pattern over buffers far larger than the last-level
        cache; the reduce pattern at the step's level shapes (P slices of the
        level's INT4 bytes + scales, back to back, and one output slice), with
        copies rotated to >= ROT_BYTES."""
        T = self.torch
        GiB = 1 << 30
        a = T.empty(2 * GiB, dtype=T.uint8, device="cuda")
        a.fill_(3)
        b = T.empty(2 * GiB, dtype=T.uint8, device="cuda")
        sink = T.zeros(16, dtype=T.uint8, device="cuda")
        A, B_, L = a.data_ptr(), b.data_ptr(), self.L
        res = {}
        us = loop_us([lambda: self._ok(L.zqp_copy(A, B_, GiB, self._st()), "copy"),
                      lambda: self._ok(L.zqp_copy(A + GiB, B_ + GiB, GiB, self._st()), "copy")], reps)
        res["copy_GBps"] = round(2 * GiB / (us * 1e-6) / 1e9, 1)
        us = loop_us([lambda: self._ok(L.zqp_read(A, 2 * GiB, sink.data_ptr(), 0x9E3779B9, self._st()), "read")], reps)
        res["read_GBps"] = round(2 * GiB / (us * 1e-6) / 1e9, 1)
        us = loop_us([lambda: self._ok(L.zqp_write(B_, 2 * GiB, 7, self._st()), "write")], reps)
        res["write_GBps"] = round(2 * GiB / (us * 1e-6) / 1e9, 1)
        us = loop_us([lambda: b[:GiB].copy_(a[:GiB])], reps)
        res["torch_copy_GBps"] = round(2 * GiB / (us * 1e-6) / 1e9, 1)
        n = 452_984_832
        streams = {}
        for P, m in ((8, n // 8), (2, n // 2), (4, n // 8), (48, n // 384), (8, n)):
            sl = (nb4(m) + 4 * nsc(m, GBLOCK) + 15) // 16 * 16
            fp = (P + 1) * sl
            nsets = max(1, min(2 * GiB // (P * sl), -(-ROT_BYTES // fp)))
            nsets = min(nsets, 2 * GiB // sl)
            runs = [lambda k=k: self._ok(L.zqp_streams(A + k * P * sl, P, sl, B_ + k * sl, self._st()), "streams")
                    for k in range(nsets)]
            us = loop_us(runs, max(reps, 2 * nsets))
            key = f"P={P} m={m}"
            streams[key] = {"GBps": round(fp / (us * 1e-6) / 1e9, 1), "us": round(us, 2), "rotated_sets": nsets}
        res["reduce_pattern"] = streams
        # the INT8 -> 16-bit dequantiser's pattern at the layer's size: n bytes
        # in, 2n out, 8 bytes loaded and 16 stored per thread
        us = loop_us([lambda: self._ok(L.zqp_expand(A, n, B_, self._st()), "expand")], reps)
        res["dequant_pattern"] = {"n": n, "GBps": round(3 * n / (us * 1e-6) / 1e9, 1), "us": round(us, 2)}
        del a, b
        T.cuda.empty_cache()
        return res


def workload_tiny(reps):
    """tiny-1024x1024: one 1024 x 1024 fp16 weight, INT8 B = 256 -> fp16; the
    fp32 gradient of the same shape from P = 2 ranks, INT4 B = 128, one level
    (rank 0's half), final dequantisation.  Latency-bound (<= 5 MB per call):
    each figure is the time per launch of back-to-back launches; then the
    whole path eagerly and as one HIP graph replay."""
    import torch

    import paper_2501_04266_amd as zq
    from paper_2501_04266_amd import workloads as wl
    n = wl.N_TINY
    w = torch.from_numpy(wl.weights(n, "f16", key=[1, wl.ROLE_WEIGHT, 0, 0])).to("cuda")
    codes = torch.empty(n, dtype=torch.int8, device="cuda")
    wsc = torch.empty(nsc(n, WBLOCK), device="cuda")
    y = torch.empty(n, dtype=torch.float16, device="cuda")
    g = [torch.from_numpy(wl.normal_f32(n, 1e-3, key=[1, wl.ROLE_OWN_GRAD if r == 0 else wl.ROLE_PEER_GRAD, 0, r]))
         .to("cuda") for r in range(2)]
    gp = torch.empty(nb4(n), dtype=torch.uint8, device="cuda")
    gs = torch.empty(nsc(n, GBLOCK), device="cuda")
    m = n // 2
    mb, ms = nb4(m), nsc(m, GBLOCK)
    pin = torch.empty(2 * mb, dtype=torch.uint8, device="cuda")
    sin = torch.empty(2 * ms, device="cuda")
    for r in range(2):      # rank r's chunk 0 arrives as slice r of rank 0's receive buffer
        zq.qgz_quantize(g[r][:m], GBLOCK, packed=pin[r * mb:(r + 1) * mb], scales=sin[r * ms:(r + 1) * ms])
    rp = torch.empty(mb, dtype=torch.uint8, device="cuda")
    rs = torch.empty(ms, device="cuda")
    gy = torch.empty(m, device="cuda")
    runs = [
        ("qwz_quantize", bytes_qwz_quant(n, 2, WBLOCK), n,
         lambda: zq.qwz_quantize(w, WBLOCK, codes=codes, scales=wsc)),
        ("qwz_dequantize", bytes_qwz_deq(n, 2, WBLOCK), n, lambda: zq.qwz_dequantize(codes, wsc, WBLOCK, y=y)),
        ("qgz_quantize", bytes_qgz_quant(n, 4, GBLOCK), n,
         lambda: zq.qgz_quantize(g[0], GBLOCK, packed=gp, scales=gs)),
        ("qgz_reduce_level P=2", bytes_reduce(2, m, GBLOCK), 2 * m,
         lambda: zq.qgz_reduce_level(pin, sin, 2, m, GBLOCK, packed_out=rp, scales_out=rs)),
        ("qgz_dequantize", bytes_qgz_deq(m, 4, GBLOCK), m, lambda: zq.qgz_dequantize(rp, rs, m, GBLOCK, y=gy)),
    ]
    figs = [call_figures(name, nb, el, loop_us([fn], reps)) for name, nb, el, fn in runs]

    # the whole path (five calls) launched eagerly against replayed from one
    # HIP graph (the calls enqueue only kernels, so they can be captured);
    # every output of a replay must equal the eager outputs bit for bit
    def path():
        for _, _, _, fn in runs:
            fn()

    path()
    torch.cuda.synchronize()
    outs = (codes, wsc, y, gp, gs, rp, rs, gy)
    want = [t.clone() for t in outs]
    eager_us = loop_us([path], reps)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        with torch.cuda.graph(graph, stream=s):
            path()
    torch.cuda.synchronize()
    for t in outs:
        t.zero_()
    graph.replay()
    torch.cuda.synchronize()
    same = all(torch.equal(a.view(torch.uint8), b.view(torch.uint8)) for a, b in zip(outs, want))
    graph_us = loop_us([graph.replay], reps)
    figs.append({"call": "whole path (5 calls)", "eager_us": round(eager_us, 2), "graph_replay_us": round(graph_us, 2),
                 "graph_bit_identical": same})
    return figs


def workload_13b(reps):
    """gpt-1.3b-layer: the GPT-1.3B-shaped layer (12 h^2, h = 2048,
    50,331,648 parameters): bf16 weight shard 1/8 -> INT8 B = 256, the
    gathered layer -> bf16; fp32 gradient -> INT4 B = 128, one P = 8 level
    (m = n/8) and its all-shares mode (m = n), the shard -> fp32.  Every
    call's inputs rotate over copies totalling >= 1.1 GB."""
    import torch

    import paper_2501_04266_amd as zq
    from paper_2501_04266_amd import workloads as wl
    np = __import__("numpy")
    n = wl.N_13B
    s, m = n // SHARD, n // 8
    w = torch.from_numpy(wl.weights(n, "bf16", key=[2, wl.ROLE_WEIGHT, 0, 0]).view(np.int16)).to("cuda").view(
        torch.bfloat16)
    codes = torch.empty(n, dtype=torch.int8, device="cuda")
    wsc = torch.empty(nsc(n, WBLOCK), device="cuda")
    zq.qwz_quantize(w, WBLOCK, codes=codes, scales=wsc)          # the gathered layer (all 8 shards)
    y = torch.empty(n, dtype=torch.bfloat16, device="cuda")
    g = torch.from_numpy(wl.normal_f32(n, 1e-3, key=[2, wl.ROLE_OWN_GRAD, 0, 0])).to("cuda")
    gp = torch.empty(nb4(n), dtype=torch.uint8, device="cuda")
    gs = torch.empty(nsc(n, GBLOCK), device="cuda")
    zq.qgz_quantize(g, GBLOCK, packed=gp, scales=gs)
    mb, ms = nb4(m), nsc(m, GBLOCK)
    pin = torch.empty(8 * mb, dtype=torch.uint8, device="cuda")
    sin = torch.empty(8 * ms, device="cuda")
    pin[:mb].copy_(gp[:mb])
    sin[:ms].copy_(gs[:ms])
    for p in range(1, 8):
        xs = torch.from_numpy(wl.normal_f32(m, 1e-3, key=[2, wl.ROLE_PEER_GRAD, 0, p])).to("cuda")
        zq.qgz_quantize(xs, GBLOCK, packed=pin[p * mb:(p + 1) * mb], scales=sin[p * ms:(p + 1) * ms])
    apin = torch.from_numpy(wl.random_bytes(8 * nb4(n), key=[2, wl.ROLE_MISC, 9, 0])).to("cuda")
    asin = torch.from_numpy(wl.uniform_f32(8 * nsc(n, GBLOCK), *wl.ALL_SHARES_SCALES, key=[2, wl.ROLE_MISC, 9, 1])).to(
        "cuda")
    U8, F32 = torch.uint8, torch.float32
    E = lambda k, dt: torch.empty(k, dtype=dt, device="cuda")
    specs = [
        ("qwz_quantize", bytes_qwz_quant(s, 2, WBLOCK), s,
         lambda i, o: zq.qwz_quantize(i[0], WBLOCK, codes=o[0], scales=o[1]), [w[:s]],
         [codes[:s], wsc[:nsc(s, WBLOCK)]]),
        ("qwz_dequantize", bytes_qwz_deq(n, 2, WBLOCK), n, lambda i, o: zq.qwz_dequantize(i[0], i[1], WBLOCK, y=o[0]),
         [codes, wsc], [y]),
        ("qgz_quantize", bytes_qgz_quant(n, 4, GBLOCK), n,
         lambda i, o: zq.qgz_quantize(i[0], GBLOCK, packed=o[0], scales=o[1]), [g], [gp, gs]),
        ("qgz_reduce_level P=8", bytes_reduce(8, m, GBLOCK), 8 * m,
         lambda i, o: zq.qgz_reduce_level(i[0], i[1], 8, m, GBLOCK, packed_out=o[0], scales_out=o[1]), [pin, sin],
         [E(mb, U8), E(ms, F32)]),
        ("qgz_reduce_level P=8 all-shares (m = n)", bytes_reduce(8, n, GBLOCK), 8 * n,
         lambda i, o: zq.qgz_reduce_level(i[0], i[1], 8, n, GBLOCK, packed_out=o[0], scales_out=o[1]), [apin, asin],
         [E(nb4(n), U8), E(nsc(n, GBLOCK), F32)]),
        ("qgz_dequantize", bytes_qgz_deq(m, 4, GBLOCK), m, lambda i, o: zq.qgz_dequantize(i[0], i[1], m, GBLOCK, y=o[0]),
         [gp[:mb], gs[:ms]], [E(m, F32)]),
    ]
    return timed_calls(specs, reps)


def workload_edge(reps):
    """outlier-edge-123456789: 123,456,789 fp32 elements (not a multiple of
    any block), 0.02 * Student-t(3) with 0.1% of them x100 and zero groups:
    INT8 B = 256 and INT4 B = 64, each quantised and dequantised to bf16.
    Inputs rotate over copies totalling >= 1.1 GB."""
    import torch

    import paper_2501_04266_amd as zq
    from paper_2501_04266_amd import workloads as wl
    n = wl.N_EDGE
    x = torch.from_numpy(wl.outlier_tensor(n, key=[5, wl.ROLE_WEIGHT, 0, 0])).to("cuda")
    c8, s8 = zq.qwz_quantize(x, 256)
    p4, s4 = zq.qgz_quantize(x, 64)
    BF = torch.bfloat16
    specs = [
        ("qwz_quantize INT8 B=256", bytes_qwz_quant(n, 4, 256), n,
         lambda i, o: zq.qwz_quantize(i[0], 256, codes=o[0], scales=o[1]), [x], [c8, s8]),
        ("qwz_dequantize INT8 -> bf16", bytes_qwz_deq(n, 2, 256), n,
         lambda i, o: zq.qwz_dequantize(i[0], i[1], 256, y=o[0]), [c8, s8],
         [torch.empty(n, dtype=BF, device="cuda")]),
        ("qgz_quantize INT4 B=64", bytes_qgz_quant(n, 4, 64), n,
         lambda i, o: zq.qgz_quantize(i[0], 64, packed=o[0], scales=o[1]), [x], [p4, s4]),
        ("qgz_dequantize INT4 -> bf16", bytes_qgz_deq(n, 2, 64), n,
         lambda i, o: zq.qgz_dequantize(i[0], i[1], n, 64, y=o[0]), [p4, s4],
         [torch.empty(n, dtype=BF, device="cuda")]),
    ]
    return timed_calls(specs, reps)


def step_call_specs(L):
    """(name, bytes, elements, fn, inputs, outputs) of each call of the step,
    on the step's own buffers."""
    zq = L.zq
    s = L.shard
    specs = [
        (lambda i, o: zq.qwz_quantize(i[0], WBLOCK, codes=o[0], scales=o[1]), [L.w[:s]],
         [L.codes[:s], L.wscales[:nsc(s, WBLOCK)]]),
        (lambda i, o: zq.qwz_dequantize(i[0], i[1], WBLOCK, y=o[0]), [L.codes, L.wscales], [L.y]),
        (lambda i, o: zq.qgz_quantize(i[0], GBLOCK, packed=o[0], scales=o[1]), [L.g], [L.gp, L.gs]),
        (lambda i, o: zq.qgz_reduce_level(i[0], i[1], 8, L.m8, GBLOCK, packed_out=o[0], scales_out=o[1]),
         list(L.d8), list(L.o8)),
        (lambda i, o: zq.qgz_dequantize(i[0], i[1], L.m8, GBLOCK, y=o[0]), list(L.o8), [L.gshard]),
    ]
    for P, m, d, o in L.chain:
        specs.append((lambda i, o_, P=P, m=m: zq.qgz_reduce_level(i[0], i[1], P, m, GBLOCK, packed_out=o_[0],
                                                                  scales_out=o_[1]), list(d), list(o)))
    P, m, d, o = L.chain[-1]
    specs.append((lambda i, o_, m=m: zq.qgz_dequantize(i[0], i[1], m, GBLOCK, y=o_[0]), list(o), [L.final]))
    return [(name, b, e, fn, ins, outs) for (name, b, e), (fn, ins, outs) in zip(L.calls, specs)]


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--settle", type=int, default=100,
                    help="steps run after the warm-up, before timing, while the GPU's clock settles")
    ap.add_argument("--dom-every", type=int, default=4,
                    help="time the dominant kernel with an event pair in every N-th step of the timed region")
    ap.add_argument("--no-cpu-baseline", action="store_true", help="skip the oracle timing and full check")
    ap.add_argument("--cpu-threads", type=int, default=0, help="oracle threads (default: all available)")
    ap.add_argument("--cpu-repeats", type=int, default=3, help="oracle repetitions of each timed call")
    ap.add_argument("--no-single-thread", action="store_true", help="skip the 1-thread oracle step")
    ap.add_argument("--steps-gemm", type=int, default=10, help="timed repetitions of the layer's GEMMs")
    ap.add_argument("--no-extras", action="store_true", help="the step only (no other workloads, ceilings or GEMMs)")
    ap.add_argument("--n", type=int, default=0, help=argparse.SUPPRESS)  # smaller layer for quick checks
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: this path runs on one GPU only (the P slices of each level are held in one "
              "GPU's HBM); --gpus must be 1", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2501_04266_amd as zq
    from paper_2501_04266_amd import workloads as wl

    if not os.path.exists(zq.LIB_PATH):
        from paper_2501_04266_amd import build as zbuild
        zbuild.build()
    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)

    def log(msg):
        print(f"[bench] {msg}", file=sys.stderr, flush=True)

    n = args.n or wl.N_20B
    L = Layer20B(n, log)
    ncalls = len(L.calls)
    for _ in range(args.warmup):
        L.step()
    torch.cuda.synchronize()
    log(f"warmup {args.warmup} done")

    # breakdown pass (not the timed region): HIP events between all calls of
    # each step; even a fence-free event between two launches costs about
    # 1.7 us of GPU time, so these figures are per call but the step time is
    # not taken here
    evs = [[TimingEvent() for _ in range(ncalls + 1)] for _ in range(args.steps)]
    for k in range(args.steps):
        L.step(evs[k])
    torch.cuda.synchronize()
    call_ms = np.array([[evs[k][i].elapsed_time(evs[k][i + 1]) for i in range(ncalls)]
                        for k in range(args.steps)])
    per_call_ms, per_call_med = call_ms.mean(axis=0), np.median(call_ms, axis=0)
    dom = max(range(ncalls), key=lambda i: per_call_ms[i])
    dom_name, dom_bytes, _ = L.calls[dom]

    # settle, right before the timed region: the clock falls for some tens of
    # milliseconds once continuous heavy work starts (also after the breakdown
    # pass, whose events leave short idle gaps), then recovers; blocks of 10
    # steps are timed to report the transient
    blocks = [min(10, args.settle - k) for k in range(0, args.settle, 10)]
    sev = [TimingEvent() for _ in range(len(blocks) + 1)]
    sev[0].record()
    for j, nb_ in enumerate(blocks):
        for _ in range(nb_):
            L.step()
        sev[j + 1].record()
    torch.cuda.synchronize()
    settle = [sev[j].elapsed_time(sev[j + 1]) / nb_ for j, nb_ in enumerate(blocks)]
    log(f"settle {args.settle} steps: " + " ".join(f"{v:.3f}" for v in settle))

    # timed region: K steps; the only events recorded are the pairs around the
    # dominant kernel in every --dom-every-th step, which give the roofline
    # figure (each pair is a barrier that costs the step a few microseconds)
    sampled = list(range(0, args.steps, max(1, args.dom_every)))
    dev = {k: [TimingEvent() for _ in range(2)] for k in sampled}
    r0, r1 = TimingEvent(), TimingEvent()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    r0.record()
    for k in range(args.steps):
        L.step(dev.get(k), around=dom)
    r1.record()
    t_enq = time.perf_counter()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    gpu_ms_per_step = r0.elapsed_time(r1) / args.steps
    enqueue_ms_per_step = (t_enq - t0) * 1e3 / args.steps
    log(f"timed {args.steps} steps: {ms_per_step:.3f} ms/step (GPU events {gpu_ms_per_step:.3f}, "
        f"host enqueue {enqueue_ms_per_step:.3f})")
    dom_ms = np.array([dev[k][0].elapsed_time(dev[k][1]) for k in sampled])

    step_bytes = sum(b for _, b, _ in L.calls)
    step_elems = sum(e for _, _, e in L.calls)
    value = step_bytes / (ms_per_step * 1e-3) / 1e9
    achieved = dom_bytes / (dom_ms.mean() * 1e-3) / 1e9
    traffic = load_traffic(dom_name)

    # per call: rotated back-to-back loops, the step's event brackets, the
    # committed trace's kernel-only duration
    kernels = timed_calls(step_call_specs(L), 40)
    for k, ms, med in zip(kernels, per_call_ms, per_call_med):
        k["us_in_step_events"] = round(ms * 1e3, 2)
        k["us_in_step_events_median"] = round(med * 1e3, 2)
        tr = load_trace(k["call"])
        if tr is not None:
            k["us_trace"] = tr
            k["pct_hbm_peak_trace"] = round(100 * k["bytes"] / (tr * 1e-6) / 1e9 / HBM_PEAK_GBPS, 1)
        valu = load_valu(k["call"])
        if valu is not None:
            k["valu"] = valu
        if k["bytes"] >= GATE_BYTES:
            k["gate_70pct"] = {"loop": k["pct_hbm_peak"] >= 70.0, "trace": (k.get("pct_hbm_peak_trace", 0) >= 70.0
                                                                          if tr is not None else None)}
    log("per-call loops done")

    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "GB/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": "gpt-20b-layer qwZ/qgZ step (h=6144, ffn=24576, n=452,984,832): "
                               "qwz shard 1/8 bf16 B=256 + gathered dequant -> bf16; qgz fp32 B=128, "
                               "P=8 level + 3-level chain P=2/4/48, final dequant -> fp32",
                   "n": n, "step_bytes": step_bytes, "step_elements": step_elems,
                   "pct_hbm_peak": round(100 * value / HBM_PEAK_GBPS, 1),
                   "elements_per_s": round(step_elems / (ms_per_step * 1e-3)),
                   "ms_per_step_gpu_events": round(gpu_ms_per_step, 4),
                   "host_enqueue_ms_per_step": round(enqueue_ms_per_step, 4),
                   "settle_steps": args.settle,
                   "settle_ms_per_step_by_10": [round(v, 4) for v in settle]},
        "roofline": {"bound": "hbm", "kernel": dom_name, "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": traffic,
                     "bytes_per_launch": dom_bytes, "us_per_launch": round(dom_ms.mean() * 1e3, 2),
                     "us_median": round(float(np.median(dom_ms)) * 1e3, 2), "launches_timed": len(sampled)},
        "kernels": kernels,
    }

    if not args.no_extras:
        extras(L, args, out, log)

    if not args.no_cpu_baseline:
        threads = args.cpu_threads or max(1, len(os.sched_getaffinity(0)))
        log(f"oracle step on {threads} threads ...")
        secs, outs = oracle_step(L, threads, args.cpu_repeats)
        bad = check_against_oracle(L, outs)
        out["cpu_baseline"] = {"value": round(step_bytes / secs / 1e9, 3), "unit": "GB/s", "cores": threads,
                               "kind": "oracle", "seconds_per_step": round(secs, 3), "cpu_model": cpu_model(),
                               "sample": f"the full step of the same workload (all calls, full sizes), each timed "
                                         f"call repeated {args.cpu_repeats}x, mean",
                               "per_call_s": dict(zip([c for c, _, _ in L.calls], outs["per_call_s"]))}
        if threads > 1 and not args.no_single_thread:
            log("oracle step on 1 thread ...")
            secs1, _ = oracle_step(L, 1, 1)
            out["cpu_baseline"]["single_thread"] = {"value": round(step_bytes / secs1 / 1e9, 3),
                                                    "seconds_per_step": round(secs1, 3)}
        out["parity"] = "bit-exact vs oracle (all step outputs)" if not bad else f"MISMATCH: {bad}"
        log(f"oracle {secs:.1f}s; parity: {out['parity']}")
    print(json.dumps(out), flush=True)


def extras(L, args, out, log):
    """The fields measured after the timed region (see the module docstring)."""
    import torch

    from paper_2501_04266_amd import workloads as wl
    zq, n = L.zq, L.n
    reps = max(args.steps, 20)

    # the other workloads, call by call
    out["workloads"] = {"tiny-1024x1024 (latency-bound)": workload_tiny(max(reps, 100)),
                        "gpt-1.3b-layer": workload_13b(reps),
                        "outlier-edge-123456789": workload_edge(reps)}
    log("workloads done")

    # bandwidth ceilings of plain access patterns (hand-written kernels)
    out["ceilings"] = Probe().ceilings()
    out["copy_ceiling_GBps"] = out["ceilings"]["copy_GBps"]
    log(f"ceilings: {out['ceilings']['copy_GBps']} GB/s copy")

    # next row: the last level fused with the final dequantisation, against the
    # two separate calls it replaces (same inputs, same outputs bit for bit)
    fused = {}
    for label, (P, m, d, o), yout in (("P=8 level + dequant", (8, L.m8, L.d8, L.o8), L.gshard),
                                      ("P=48 level + dequant", L.chain[-1], L.final)):
        sep_fn = lambda i, o_, P=P, m=m, yout=yout: (
            zq.qgz_reduce_level(i[0], i[1], P, m, GBLOCK, packed_out=o_[0], scales_out=o_[1]),
            zq.qgz_dequantize(o_[0], o_[1], m, GBLOCK, y=o_[2]))
        fus_fn = lambda i, o_, P=P, m=m: zq.qgz_reduce_dequantize(i[0], i[1], P, m, GBLOCK, y=o_[2])
        outs = [o[0], o[1], yout]
        t_sep = loop_us(rotation_runs(sep_fn, list(d), outs), reps)
        t_fus = loop_us(rotation_runs(fus_fn, list(d), outs), reps)
        fused_bytes = P * (nb4(m) + 4 * nsc(m, GBLOCK)) + 4 * m
        fused[label] = {"separate_us": round(t_sep, 2), "fused_us": round(t_fus, 2), "fused_bytes": fused_bytes,
                        "fused_GBps": round(fused_bytes / (t_fus * 1e-6) / 1e9, 1)}
        torch.cuda.empty_cache()
    out["fused_last_level"] = fused

    # all-shares mode of the P=8 level: 8 slices of the whole layer (m = n),
    # random INT4 codes and scales, 2.17 GB per launch (beyond the cache):
    # the first launches after the legs before it, then (the headline figure)
    # the same after ALL_SHARES_SETTLE_S seconds of launches, once the clock
    # has recovered from the dip that sustained reduce work causes
    pin = torch.from_numpy(wl.random_bytes(8 * nb4(n), key=[3, wl.ROLE_MISC, 9, 0])).to("cuda")
    sin = torch.from_numpy(wl.uniform_f32(8 * nsc(n, GBLOCK), *wl.ALL_SHARES_SCALES,
                                          key=[3, wl.ROLE_MISC, 9, 1])).to("cuda")
    aop = torch.empty(nb4(n), dtype=torch.uint8, device="cuda")
    aos = torch.empty(nsc(n, GBLOCK), dtype=torch.float32, device="cuda")
    allsh = lambda: zq.qgz_reduce_level(pin, sin, 8, n, GBLOCK, packed_out=aop, scales_out=aos)
    first_us = loop_us([allsh], reps, warm=0)           # right after the lighter legs before it
    t_end = time.perf_counter() + ALL_SHARES_SETTLE_S    # then the clock's dip and recovery
    while time.perf_counter() < t_end:
        for _ in range(8):
            allsh()
        torch.cuda.synchronize()
    as_us = loop_us([allsh], reps, warm=0)
    as_bytes = bytes_reduce(8, n, GBLOCK)
    out["all_shares"] = {"qgz_reduce_level P=8 m=n us": round(as_us, 2), "bytes": as_bytes,
                         "GBps": round(as_bytes / (as_us * 1e-6) / 1e9, 1),
                         "pct_hbm_peak": round(100 * as_bytes / (as_us * 1e-6) / 1e9 / HBM_PEAK_GBPS, 1),
                         "settle_s": ALL_SHARES_SETTLE_S,
                         "first_launches_us": round(first_us, 2),
                         "first_launches_GBps": round(as_bytes / (first_us * 1e-6) / 1e9, 1)}
    del pin, sin, aop, aos
    torch.cuda.empty_cache()

    # next row: the P=8 level reading its slices in place from 8 separate
    # buffers through device pointer tables (how a receiver would read peers'
    # send buffers mapped over xGMI) against the contiguous receive buffer;
    # both over rotated copies
    mb8, ms8 = nb4(L.m8), nsc(L.m8, GBLOCK)
    nsets = 4
    gsets = []
    for _ in range(nsets):
        gp_sl = [L.d8[0][p * mb8:(p + 1) * mb8].clone() for p in range(8)]
        gs_sl = [L.d8[1][p * ms8:(p + 1) * ms8].clone() for p in range(8)]
        gsets.append((gp_sl, gs_sl, zq.gather_tables(gp_sl, gs_sl)))
    csets = [(L.d8[0].clone(), L.d8[1].clone()) for _ in range(nsets)]
    go = (torch.empty(mb8, dtype=torch.uint8, device="cuda"), torch.empty(ms8, dtype=torch.float32, device="cuda"))
    co = (torch.empty(mb8, dtype=torch.uint8, device="cuda"), torch.empty(ms8, dtype=torch.float32, device="cuda"))
    g_runs = [lambda s=s: zq.qgz_reduce_level_gather(s[0], s[1], L.m8, GBLOCK, packed_out=go[0], scales_out=go[1],
                                                     tables=s[2]) for s in gsets]
    c_runs = [lambda s=s: zq.qgz_reduce_level(s[0], s[1], 8, L.m8, GBLOCK, packed_out=co[0], scales_out=co[1])
              for s in csets]
    t_c, t_g = loop_us(c_runs, reps), loop_us(g_runs, reps)
    same = bool(torch.equal(go[0], co[0]) and torch.equal(go[1], co[1]))
    out["reduce_gather"] = {"P=8 level contiguous us": round(t_c, 2), "P=8 level gather us": round(t_g, 2),
                            "gather_GBps": round(bytes_reduce(8, L.m8, GBLOCK) / (t_g * 1e-6) / 1e9, 1),
                            "bit_identical": same, "rotated_sets": nsets}
    del gsets, csets
    torch.cuda.empty_cache()

    # next row: the degree-2 weight partition (1/2 shard quantised into its slot
    # of the gathered buffer; the dequantisation of the gathered layer is the
    # same call as in the step)
    half = n // 2
    sd2_us = loop_us([lambda: zq.qwz_quantize(L.w[:half], WBLOCK, codes=L.codes[:half],
                                              scales=L.wscales[:nsc(half, WBLOCK)])], reps)
    sd2_bytes = bytes_qwz_quant(half, 2, WBLOCK)
    out["sec_degree_2"] = {"qwz_quantize half-shard us": round(sd2_us, 2), "bytes": sd2_bytes,
                           "GBps": round(sd2_bytes / (sd2_us * 1e-6) / 1e9, 1)}

    # next row: the layer's forward GEMMs with the gathered INT8 weight
    # dequantised on load (qwz_dequant_gemm), 8192 tokens of bf16 activations,
    # against dequantising the layer to bf16 and running torch's GEMM on it
    out["dequant_gemm"] = gemm_figures(L, args.steps_gemm, log)


if __name__ == "__main__":
    main()
