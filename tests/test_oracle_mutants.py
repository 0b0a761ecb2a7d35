"""Mutation test of the oracle's pins (CPU only).

Each mutant is a copy of oracle/zq_oracle.c with one plausible mistake
planted (a wrong rounding rule, divide instead of reciprocal multiply, a
dropped flush threshold, reversed slice order, swapped nibbles, a transposed
scale index, truncating narrowing, ...).  The copy is compiled into a
temporary library and the pin checks of tests/pin_checks.py run against it in
a child process; every mutant must fail at least one pin.  The real oracle
must pass them all.
"""
import json
import os
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

import pytest

from oracle import build as obuild

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# (name, [(old, new), ...], extra compiler flags)
MUTANTS = [
    ("ties-away", [("float k = nearbyintf(t);", "float k = roundf(t);")], []),
    ("divide-by-scale", [("float t = v[i] * r;", "float t = v[i] / s;")], []),
    ("no-flush-threshold", [("if (a < 0x1p-119f) {", "if (a <= 0.0f) {")], []),
    ("scale-qmax-plus-1", [("float s = a / (float)qmax;", "float s = a / (float)(qmax + 1);")], []),
    ("signed-absmax", [("if (m > a) a = m;", "if (m > a) a = v[i];")], []),
    ("reverse-slice-order", [("for (int32_t p = 0; p < P; ++p) {", "for (int32_t p = P - 1; p >= 0; --p) {")], []),
    ("transposed-scale-index", [("scales_in[(int64_t)p * nb + b]", "scales_in[(int64_t)b * P + p]")], []),
    ("swapped-nibbles", [("(uint8_t)((q[i] & 0x0f) | ((q[i + 1] & 0x0f) << 4))",
                          "(uint8_t)(((q[i] & 0x0f) << 4) | (q[i + 1] & 0x0f))")], []),
    ("nibble-sign", [("return v >= 8 ? v - 16 : v;", "return v >= 7 ? v - 16 : v;")], []),
    ("int8-unsigned", [("float prod = (float)codes[i] * scales[i / block];",
                        "float prod = (float)(uint8_t)codes[i] * scales[i / block];")], []),
    ("dequant-block-off-by-one", [("float prod = (float)codes[i] * scales[i / block];",
                                   "float prod = (float)codes[i] * scales[(i + 1) / block];")], []),
    ("bf16-truncate", [("if (dropped > 0x8000u || (dropped == 0x8000u && (upper & 1u))) upper += 1u;", "")], []),
    ("f16-subnormal-exponent", [("if (e == 0) v = ldexpf((float)m, -24);", "if (e == 0) v = ldexpf((float)m, -25);")], []),
    ("f16-ties-away", [("double k = nearbyint((double)a / spacing);", "double k = floor((double)a / spacing + 0.5);")], []),
    ("fused-multiply-add", [], ["-ffp-contract=fast", "-mfma"]),
]


def _run_checks(lib_path):
    env = dict(os.environ, ZQ_ORACLE_LIB=lib_path, OMP_NUM_THREADS="1")
    r = subprocess.run([sys.executable, "-m", "tests.pin_checks", "--first"], cwd=ROOT, env=env,
                       capture_output=True, text=True, timeout=600)
    if r.returncode != 0:
        return ["child-crashed"]
    return json.loads(r.stdout.strip().splitlines()[-1])


def _mutant(tmp, name, subs, flags):
    src = open(obuild.SRC).read()
    for old, new in subs:
        assert src.count(old) >= 1, f"mutant {name}: pattern not found: {old}"
        src = src.replace(old, new)
    path = os.path.join(tmp, f"{name}.c")
    open(path, "w").write(src)
    lib = os.path.join(tmp, f"lib{name}.so")
    obuild.build(src=path, out=lib, extra=flags + ["-w"])
    return name, _run_checks(lib)


def test_oracle_passes_all_pins():
    from tests import pin_checks
    assert pin_checks.run_all() == []


@pytest.mark.slow
def test_every_mutant_is_caught():
    with tempfile.TemporaryDirectory() as tmp:
        with ThreadPoolExecutor(max(1, min(8, os.cpu_count() or 1))) as ex:
            results = list(ex.map(lambda m: _mutant(tmp, *m), MUTANTS))
    survivors = [name for name, failed in results if not failed]
    assert not survivors, f"mutants not caught by any pin: {survivors}"


# Mistakes planted in the oracle's level composition (oracle.chain), which is
# Python: each is applied to the function's source and the brute-force chain
# pin must reject the result (a crash also counts as detection; every mutant
# here keeps the slice sizes right, except the stale level size).
CHAIN_MUTANTS = [
    ("own-chunk-always-0", [("own_chunk_p = cur_p[rank * mb:(rank + 1) * mb]", "own_chunk_p = cur_p[0:mb]"),
                            ("own_chunk_s = cur_s[rank * nbm:(rank + 1) * nbm]", "own_chunk_s = cur_s[0:nbm]")]),
    ("scale-offset-in-chunks", [("own_chunk_s = cur_s[rank * nbm:(rank + 1) * nbm]",
                                 "own_chunk_s = cur_s[rank:rank + nbm]")]),
    ("next-chunk", [("own_chunk_p = cur_p[rank * mb:(rank + 1) * mb]",
                     "own_chunk_p = cur_p[(rank + 1) % P * mb:((rank + 1) % P + 1) * mb]"),
                    ("own_chunk_s = cur_s[rank * nbm:(rank + 1) * nbm]",
                     "own_chunk_s = cur_s[(rank + 1) % P * nbm:((rank + 1) % P + 1) * nbm]")]),
    ("own-slice-first", [("for p in range(P):\n            if p == rank:",
                          "slices_p.append(own_chunk_p)\n        slices_s.append(own_chunk_s)\n"
                          "        for p in range(P):\n            if p == rank:\n                continue\n"
                          "            if False:")]),
    ("stale-level-size", [("        cur_m = m\n", "")]),
]


def _mutated_chain(subs):
    import inspect
    import textwrap

    import numpy as np

    import oracle
    src = textwrap.dedent(inspect.getsource(oracle.chain))
    for old, new in subs:
        assert src.count(old) == 1, f"chain mutant pattern not found: {old}"
        src = src.replace(old, new)
    ns = {"np": np, "num_scales": oracle.num_scales, "int4_bytes": oracle.int4_bytes,
          "qgz_reduce_level": oracle.qgz_reduce_level}
    exec(compile(src, "<chain mutant>", "exec"), ns)
    return ns["chain"]


def test_chain_passes_pin():
    from tests import pin_checks
    pin_checks.check_brute_chain()


@pytest.mark.parametrize("name,subs", CHAIN_MUTANTS, ids=[m[0] for m in CHAIN_MUTANTS])
def test_every_chain_mutant_is_caught(name, subs):
    from tests import pin_checks
    fn = _mutated_chain(subs)
    with pytest.raises(Exception):
        pin_checks.check_brute_chain(chain_fn=fn)
