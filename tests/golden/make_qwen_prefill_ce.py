"""Write tests/golden/qwen_prefill_ce_v1.txt: the oracle's per-token CE of the
Qwen3-8B-shaped prefill workload (V=151936, d=4096, 4096 tokens, Zipf(1.1)
targets) and its mean, for the full-size GPU parity test.

Calls only the CPU oracle (fp64, dense head formed in row chunks) and the
seeded input generators; nothing here comes from the HIP library.  The file
also records SHA-256 digests of the generated x bits and targets, so a test
run on another machine detects a generator that drew different inputs.

Usage: python tests/golden/make_qwen_prefill_ce.py   (a few CPU minutes)
"""
from __future__ import annotations

import hashlib
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from oracle import head as ohead  # noqa: E402
from synth import CONFIGS, make_head, make_targets, make_x  # noqa: E402

OUT = os.path.join(HERE, "qwen_prefill_ce_v1.txt")
TOKEN_CHUNK = 512


def digests(x_bits: np.ndarray, y: np.ndarray):
    return (hashlib.sha256(np.ascontiguousarray(x_bits).tobytes()).hexdigest(),
            hashlib.sha256(np.ascontiguousarray(y.astype(np.int32)).tobytes()).hexdigest())


def main():
    cfg = "qwen_prefill"
    M = CONFIGS[cfg]["Ms"][0]
    h = make_head("qwen_decode")
    x = make_x(cfg, M)
    y = make_targets(cfg, M)
    ce = np.empty(M)
    t0 = time.time()
    for m0 in range(0, M, TOKEN_CHUNK):
        m1 = min(M, m0 + TOKEN_CHUNK)
        ce[m0:m1] = ohead.cross_entropy(ohead.logits(h, x[m0:m1]), y[m0:m1])
        print(f"tokens {m0}..{m1 - 1}: {time.time() - t0:.0f} s", flush=True)
    hx, hy = digests(x, y)
    with open(OUT, "w") as f:
        f.write("# Oracle (fp64) per-token cross-entropy, natural log, of the Qwen3-8B-shaped\n"
                "# prefill workload: packed head V=151936 d=4096 g=128 r_c=64 r_r=32 (fp16\n"
                "# scales), 4096 anisotropic bf16 tokens, Zipf(1.1) targets.\n"
                "# Written by tests/golden/make_qwen_prefill_ce.py (CPU oracle only).\n")
        f.write(f"x_sha256: {hx}\n")
        f.write(f"targets_sha256: {hy}\n")
        f.write(f"tokens: {M}\n")
        f.write(f"mean_ce: {float(np.mean(ce))!r}\n")
        for v in ce:
            f.write(f"{float(v)!r}\n")
    print(f"wrote {OUT}: mean CE {np.mean(ce):.6f} in {time.time() - t0:.0f} s")


if __name__ == "__main__":
    main()
