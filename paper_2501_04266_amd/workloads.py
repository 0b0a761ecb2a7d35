"""Seeded synthetic inputs for the qwZ / qgZ path (host numpy arrays).

This module only draws random numbers and casts them to the storage dtype;
it holds none of the method's arithmetic.  Both the HIP path (via upload)
and the CPU oracle consume exactly these arrays.

Shapes follow the paper's workloads: GPT-NeoX-20B (hidden 6144, FFN 24576,
cited in the Discussion) and a GPT-1.3B-shaped layer (hidden 2048, FFN 8192);
one transformer layer's flat parameter buffer is QKV (3h*h) + attention out
(h*h) + FC1 (4h*h) + FC2 (4h*h) = 12 h^2 elements.  Weights are N(0, 0.02)
drawn in float32 and rounded to nearest-even into fp16/bf16; gradients are
float32 N(0, 1e-3).  The paper trains on the Pile web subset with real
weights; none of that is needed or used -- these synthetic tensors stand in.

Every array is generated in fixed 4 Mi-element chunks, chunk c seeded by
SeedSequence(key + [c]) with PCG64, so the values do not depend on how many
threads generate them.  Keys are [config, role, level, slice].
"""
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

CHUNK = 1 << 22
ROLE_WEIGHT, ROLE_OWN_GRAD, ROLE_PEER_GRAD, ROLE_MISC = 0, 1, 2, 3


def layer_params(h):
    """Elements in one GPT layer's flat parameter buffer: 12 h^2."""
    return 3 * h * h + h * h + 4 * h * h + 4 * h * h


def _threads():
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _fill(out, key, draw):
    n = out.size

    def work(c):
        g = np.random.Generator(np.random.PCG64(np.random.SeedSequence(list(key) + [c])))
        s = c * CHUNK
        draw(g, out[s:min(n, s + CHUNK)])

    nchunks = (n + CHUNK - 1) // CHUNK
    if nchunks <= 1:
        for c in range(nchunks):
            work(c)
    else:
        with ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(work, range(nchunks)))
    return out


def normal_f32(n, std, key):
    """float32 N(0, std^2), n elements, deterministic in `key`."""
    out = np.empty(n, np.float32)

    def draw(g, o):
        g.standard_normal(o.size, dtype=np.float32, out=o)
        o *= np.float32(std)

    return _fill(out, key, draw)


def random_bytes(nbytes, key):
    """Uniform random bytes (uint8), deterministic in `key`.  As packed INT4
    slices these are codes uniform over all 16 nibble values."""
    out = np.empty(nbytes, np.uint8)

    def draw(g, o):
        o[:] = np.frombuffer(g.bytes(o.size), np.uint8)

    return _fill(out, key, draw)


def uniform_f32(n, lo, hi, key):
    """float32 uniform in [lo, hi), n elements, deterministic in `key`."""
    out = np.empty(n, np.float32)

    def draw(g, o):
        g.random(o.size, dtype=np.float32, out=o)
        o *= np.float32(hi - lo)
        o += np.float32(lo)

    return _fill(out, key, draw)


def to_storage(x32, dtype):
    """Round a float32 array to the storage dtype, nearest-even.
    Returns float32 / float16 arrays, or uint16 bit patterns for bf16."""
    if dtype == "f32":
        return x32
    if dtype == "f16":
        return x32.astype(np.float16)
    if dtype == "bf16":
        import torch
        t = torch.from_numpy(x32).to(torch.bfloat16)
        return t.view(torch.int16).numpy().view(np.uint16)
    raise ValueError(dtype)


def weights(n, dtype, key, std=0.02):
    return to_storage(normal_f32(n, std, key), dtype)


def outlier_tensor(n, key, block_zero=256, df=3.0, scale=0.02, outlier_frac=1e-3,
                   outlier_mult=100.0, zero_group_frac=1e-2):
    """Stress tensor: scale * Student-t(df); a fraction `outlier_frac` of the
    indices (uniform, without replacement) multiplied by `outlier_mult`;
    `zero_group_frac` of the block_zero-aligned groups, plus group 0, set to
    0.0.  The final partial group (when n is not a multiple of block_zero) is
    never zeroed."""
    out = np.empty(n, np.float32)

    def draw(g, o):
        o[:] = g.standard_t(df, o.size).astype(np.float32)
        o *= np.float32(scale)

    _fill(out, key, draw)
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence(list(key) + [1 << 30])))
    k = int(round(n * outlier_frac))
    idx = g.choice(n, size=k, replace=False)
    out[idx] *= np.float32(outlier_mult)
    ngroups = n // block_zero
    kz = int(round(ngroups * zero_group_frac))
    groups = g.choice(ngroups, size=kz, replace=False) if ngroups else np.empty(0, np.int64)
    groups = np.unique(np.concatenate([groups, [0]])) if ngroups else groups
    for gi in groups:
        out[gi * block_zero:(gi + 1) * block_zero] = 0.0
    return out


# --------------------------------------------------------------------------
# The five workloads.  Sizes are per rank (one GPU's share).
# --------------------------------------------------------------------------
N_TINY = 1024 * 1024
N_13B = layer_params(2048)      # 50,331,648
N_20B = layer_params(6144)      # 452,984,832
N_EDGE = 123_456_789
# scales of the random all-shares slices: the range of absmax/7 over blocks of
# 128 elements of an N(0, 1e-3) gradient is about [3e-4, 8e-4]
ALL_SHARES_SCALES = (2e-4, 1e-3)

# the five workloads, by name: sizes, storage types, blocks, shard degree,
# the weight dequantisation output, and the fan-ins of the gradient levels
WORKLOADS = {
    "tiny-1024x1024": dict(n=N_TINY, wdtype="f16", wblock=256, shard=1, qwz_out="f16", gblock=128, fanins=[2],
                           gout="f32"),
    "gpt-1.3b-layer": dict(n=N_13B, wdtype="bf16", wblock=256, shard=8, qwz_out="bf16", gblock=128, fanins=[8],
                           gout="f32"),
    "gpt-20b-layer": dict(n=N_20B, wdtype="bf16", wblock=256, shard=8, qwz_out="bf16", gblock=128, fanins=[8],
                          gout="f32"),
    "gpt-20b-3level": dict(n=N_20B, wdtype=None, wblock=None, shard=None, qwz_out=None, gblock=128,
                           fanins=[2, 4, 48], gout="f32"),
    "outlier-edge-123456789": dict(n=N_EDGE, wdtype="f32", wblock=256, shard=1, qwz_out="bf16", gblock=64, fanins=[],
                                   gout="bf16"),
}
