"""Loaders for the hand-written fixtures under tests/golden/."""
from __future__ import annotations

import json
import os
import types

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def layout_cases():
    """[(bytes uint8[4], codes int[8])] from int4_layout_v1.txt."""
    out = []
    with open(os.path.join(GOLDEN, "int4_layout_v1.txt")) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            lhs, rhs = line.split("->")
            b = np.array([int(t, 16) for t in lhs.split()], dtype=np.uint8)
            c = np.array([int(t) for t in rhs.split()], dtype=np.int64)
            out.append((b, c))
    return out


def worked_head():
    """(head, x_bf16_bits [3, 64], expected logits [3, 2], targets [3])."""
    with open(os.path.join(GOLDEN, "worked_head_v1.json")) as f:
        j = json.load(f)
    V, d = j["V"], j["d"]
    rows = j["res_codes_hex"]
    codes = np.array([list(bytes.fromhex(rows[0] + rows[1])),
                      list(bytes.fromhex(rows[2] + rows[3]))], dtype=np.uint8)
    h = types.SimpleNamespace(V=V, d=d, g=j["g"], rc=j["rc"], rr=j["rr"],
                              gV=j["gV"], gB=j["gB"])
    h.res_codes = codes
    h.res_scales = np.array(j["res_scales"], dtype=np.float16)
    h.core_u = np.array(j["core_u"], dtype=np.int8)
    h.core_u_scale = np.array(j["core_u_scale"], dtype=np.float16)
    h.core_v = np.ones((1, d), dtype=np.int8)
    h.core_v_scale = np.array(j["core_v_scale"], dtype=np.float16)
    h.corr_a = np.array(j["corr_a"], dtype=np.int8)
    h.corr_a_scale = np.array(j["corr_a_scale"], dtype=np.float16)
    cb = np.zeros((1, d), dtype=np.int8)
    cb[0, :32] = 1
    h.corr_b = cb
    h.corr_b_scale = np.array(j["corr_b_scale"], dtype=np.float16)
    one, half = 0x3F80, 0x3F00                  # bf16 bit patterns of 1.0, 0.5
    x = np.zeros((3, d), dtype=np.uint16)
    x[0, :32] = one
    x[0, 32:] = half
    x[1, 33] = one
    x[2, 1] = one
    return h, x, np.array(j["logits"]), np.array(j["targets"], dtype=np.int32)


def paper_metric_rows():
    rows = {}
    with open(os.path.join(GOLDEN, "paper_printed_metrics.txt")) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line:
                t = line.split()
                rows[t[0]] = dict(zip(("ratio", "ce", "dce", "ppl", "rel"),
                                      map(float, t[1:])))
    return rows


def paper_storage_rows():
    rows = {}
    with open(os.path.join(GOLDEN, "paper_storage.txt")) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line:
                t = line.split()
                rows[t[0]] = dict(V=int(t[1]), D=int(t[2]), dense=float(t[3]),
                                  packed=float(t[4]), ratio=float(t[5]))
    return rows
