"""Host-side parts of bench.py, on the CPU: the refusal of more than one GPU,
the algorithmic byte counts that the reported value and roofline are computed
from (the GPT-20B layer's step), and the gating of the committed PMC summaries
on the hash of the kernel sources they were taken on."""
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
N = 452_984_832  # the GPT-20B layer: 12 h^2, h = 6144


def test_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=300)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_step_algorithmic_bytes():
    calls = [
        bench.bytes_qwz_quant(N // 8, 2, 256),       # bf16 shard -> INT8, B = 256
        bench.bytes_qwz_deq(N, 2, 256),              # gathered layer -> bf16
        bench.bytes_qgz_quant(N, 4, 128),            # fp32 gradient -> INT4, B = 128
        bench.bytes_reduce(8, N // 8, 128),          # one P = 8 level
        bench.bytes_qgz_deq(N // 8, 4, 128),         # its shard -> fp32
        bench.bytes_reduce(2, N // 2, 128),          # chain: P = 2, 4, 48
        bench.bytes_reduce(4, N // 8, 128),
        bench.bytes_reduce(48, N // 384, 128),
        bench.bytes_qgz_deq(N // 384, 4, 128),       # final shard -> fp32
    ]
    assert calls == [170_754_048, 1_366_032_384, 2_052_587_520, 270_729_216, 256_573_440, 360_972_288,
                     150_405_120, 30_707_712, 5_345_280]
    assert sum(calls) == 4_664_107_008
    # odd sizes: the last INT4 byte and the last partial block count whole
    assert bench.bytes_qgz_quant(123_456_789, 4, 64) == 123_456_789 * 4 + 61_728_395 + 4 * 1_929_013
    assert bench.bytes_reduce(3, 1001, 128) == 4 * (501 + 4 * 8)


def _profile(tmp_path, name, text):
    p = tmp_path / name
    p.write_text(text)
    return str(p)


def test_pmc_summaries_are_used_only_for_the_sources_they_were_taken_on(tmp_path, monkeypatch):
    traffic = _profile(tmp_path, "traffic.txt",
                       "# kernel source sha256[:16]: 0123456789abcdef\n"
                       "call fetch KiB write KiB traffic B algorithmic B ratio\n"
                       "qgz_quantize 884751.5 235008.0 2052576064 2052587520 1.000\n"
                       "qgz_reduce_level P=8 117901.5 29376.0 271537539 270729216 1.003\n")
    valu = _profile(tmp_path, "valu.txt",
                    "# kernel source sha256[:16]: 0123456789abcdef\n"
                    "qgz_quantize 135806976 19.188 718849 0.748 2.32\n")
    monkeypatch.setattr(bench, "TRAFFIC_PROFILE", traffic)
    monkeypatch.setattr(bench, "VALU_PROFILE", valu)
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: "0123456789abcdef")
    assert bench.load_traffic("qgz_quantize") == 2_052_576_064
    assert bench.load_traffic("qgz_reduce_level P=8") == 271_537_539
    assert bench.load_traffic("qgz_reduce_level P=4") is None
    assert bench.load_valu("qgz_quantize") == {"valu_insts_per_elem": 19.188, "valu_busy": 0.748}
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: "fedcba9876543210")
    assert bench.load_traffic("qgz_quantize") is None
    assert bench.load_valu("qgz_quantize") is None


def test_source_hash_covers_the_codec_sources():
    names = {os.path.basename(p) for p in bench.KERNEL_SOURCES}
    assert names == {"zq_kernels.hip", "zq_internal.h", "zq_device.h", "zq_host.h", "zq_api.hip"}
    assert all(os.path.exists(p) for p in bench.KERNEL_SOURCES)
    assert len(bench.kernel_source_hash()) == 16


def test_rotation_covers_the_cache_and_binds_separate_buffers():
    import torch
    x = torch.zeros(1000, dtype=torch.uint8)
    y = torch.zeros(1000, dtype=torch.uint8)
    seen = []
    runs = bench.rotation_runs(lambda i, o: seen.append((i[0].data_ptr(), o[0].data_ptr())), [x], [y],
                               footprint=bench.ROT_BYTES // 3 + 1)
    assert len(runs) == 3
    for r in runs:
        r()
    assert seen[0] == (x.data_ptr(), y.data_ptr())
    assert len({a for a, _ in seen}) == 3 and len({b for _, b in seen}) == 3
    assert len(bench.rotation_runs(lambda i, o: None, [x], [y], footprint=2 * bench.ROT_BYTES)) == 1


def test_trace_summary_is_used_only_for_the_sources_it_was_taken_on(tmp_path, monkeypatch):
    trace = _profile(tmp_path, "trace.txt",
                     "# kernel source sha256[:16]: 0123456789abcdef\n"
                     "call  kernel  grid  trace avg us  min  max  event us\n"
                     "qgz_reduce_level P=8  k_reduce_p<128, 32, 8, 1, -1, false>  1769472  45.10  44.00  47.00  50.20\n"
                     "qgz_reduce_level P=48  k_reduce<128, 8, 16, 1, false, -1, false>  147456  12.24  11.60  14.40  17.10\n")
    monkeypatch.setattr(bench, "TRACE_PROFILE", trace)
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: "0123456789abcdef")
    assert bench.load_trace("qgz_reduce_level P=8") == 45.10
    assert bench.load_trace("qgz_reduce_level P=48") == 12.24
    assert bench.load_trace("qgz_reduce_level P=4") is None
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: "fedcba9876543210")
    assert bench.load_trace("qgz_reduce_level P=8") is None


def test_call_figures():
    f = bench.call_figures("x", 8_000_000_000, 1_000_000_000, 1_000.0)
    assert f["GBps"] == 8000.0 and f["pct_hbm_peak"] == 100.0 and f["Gelem_per_s"] == 1000.0


def test_timing_event_binds_the_hip_runtime_torch_loaded():
    # resolves the four event calls in the HIP runtime of this process (no
    # GPU call is made: creating an event needs a device)
    hip = bench.TimingEvent._runtime()
    for name in ("hipEventCreateWithFlags", "hipEventRecord", "hipEventElapsedTime", "hipEventDestroy"):
        assert getattr(hip, name).restype is not None
    maps = [ln.split()[-1] for ln in open("/proc/self/maps") if "libamdhip64.so" in ln]
    assert maps and hip._name == maps[0]
    assert bench.HIP_EVENT_DISABLE_SYSTEM_FENCE == 0x20000000


def test_ceiling_library_exports_what_the_bench_binds():
    # symbols only: loading the library launches nothing
    import ctypes

    from paper_2501_04266_amd import build as zbuild
    if not os.path.exists(zbuild.PROBE_LIB):
        import pytest
        pytest.skip("libzq_probe.so is not built")
    lib = ctypes.CDLL(zbuild.PROBE_LIB)
    for name in ("zqp_copy", "zqp_read", "zqp_write", "zqp_streams", "zqp_expand"):
        assert hasattr(lib, name), name
