"""CPU tests of bench.py's host logic: the one-GPU rule, the algorithmic
byte and flop counts its roofline figures divide by, and the committed HBM
traffic summary it reads."""
from __future__ import annotations

import os
import re
import subprocess
import sys
import types

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def _qwen():
    # the Qwen3-8B-shaped head's sizes (no arrays needed for the counts)
    return types.SimpleNamespace(V=151936, d=4096, g=128, rc=64, rr=32)


@pytest.mark.parametrize("argv,env", [(["--gpus", "2"], {}), ([], {"WORLD_SIZE": "8"})])
def test_more_than_one_gpu_is_refused(argv, env):
    """More than one GPU is refused: the bench exits with status 2
    and says so, before touching torch or a device."""
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *argv],
                       env={**os.environ, **env}, capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_mfma_algorithmic_flops_at_prefill_shape():
    """2 M V (d + r_c + r_r) at M = 4096 on the Qwen shape: 5.2176e12."""
    f = bench.mfma_algorithmic_flops(_qwen(), 4096)
    assert f == 2 * 4096 * 151936 * (4096 + 64 + 32)
    assert abs(f - 5.2176e12) / 5.2176e12 < 1e-4


def test_decode_algorithmic_bytes_at_decode_shape():
    """Packed head once + x (bf16) + fp32 logits; at the Qwen shape and
    M = 1 that is 337,091,776 B."""
    q = _qwen()
    assert bench.decode_algorithmic_bytes(336475840, q, 1) == 337091776
    assert bench.decode_algorithmic_bytes(10, q, 3) == 10 + 3 * 4096 * 2 + 3 * 151936 * 4


def test_bench_byte_count_is_the_librarys():
    """The bench divides by archead_packed_bytes of the head's descriptor;
    the oracle's independent count agrees (the cross-check the bench no
    longer needs at run time)."""
    from oracle.bytes import head_bytes
    from paper_2608_02703_amd import archead as ab
    from synth import make_head
    L = ab.host_lib()
    for scales in ("f16", "u8"):
        h = make_head("tiny", scales=scales)
        desc = ab.Desc.make(h.V, h.d, h.g, h.rc, h.rr, h.gV, h.gB,
                            scale_dtype=ab.U8 if scales == "u8" else ab.F16)
        ph = types.SimpleNamespace(desc=desc)
        import unittest.mock as um
        with um.patch("paper_2608_02703_amd.archead.lib", lambda: L):
            assert bench.lib_packed_bytes(ph) == head_bytes(h)


def test_trace_summary_takes_the_last_dispatches(tmp_path, capsys):
    """--trace-summary: per kernel, the last N dispatches of a rocprofv3
    kernel-trace CSV (warm-up dispatches excluded), median and mean in us."""
    import json
    rows = ["Kernel_Name,Start_Timestamp,End_Timestamp"]
    t = 0
    for i in range(10):             # 10 warm-up dispatches of 90 us, then 5 of 50 us
        dur = 90000 if i < 10 else 0
        rows.append(f"k_a,{t},{t + dur}")
        t += 100000
    for i in range(5):
        rows.append(f"k_a,{t},{t + 50000 + 1000 * i}")
        t += 100000
    rows.append(f"k_b,{t},{t + 7000}")
    p = tmp_path / "kt.csv"
    p.write_text("\n".join(rows) + "\n")
    bench.trace_summary(str(p), 5, "k_a")
    out = [json.loads(line) for line in capsys.readouterr().out.splitlines()]
    assert len(out) == 1 and out[0]["kernel"] == "k_a"
    assert out[0]["dispatches"] == 15 and out[0]["summarised"] == 5
    assert out[0]["median_us"] == 52.0 and out[0]["mean_us"] == 52.0


def test_traffic_summary_is_well_formed():
    """The committed counter summary names its per-launch bytes and the
    SHA-256 of the kernel source it was taken on; bench.py reports the
    bytes only while that SHA matches (else null)."""
    text = open(bench.TRAFFIC_FILE).read()
    t = re.search(r"traffic_bytes_per_launch:\s*([0-9]+)", text)
    h = re.search(r"source_sha256:\s*([0-9a-f]{64})", text)
    assert t and h
    got = bench.measured_traffic()
    if h.group(1) == bench.source_sha256():
        assert got == int(t.group(1))
        # within a few percent of the algorithmic bytes (no re-reads)
        assert 1.0 <= got / 337091776 < 1.1
    else:
        assert got is None
