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
    from synth import make_head
    h = make_head("tiny")
    from oracle.bytes import head_bytes
    assert bench.decode_algorithmic_bytes(h, 3) == head_bytes(h) + 3 * h.d * 2 + 3 * h.V * 4
    # the Qwen figure quoted beside the traffic counters
    assert 336475840 + 4096 * 2 + 151936 * 4 == 337091776


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
