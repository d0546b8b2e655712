"""GPU parity of every tile layout of the many-token kernel, through the C
ABI: 64-row tiles of 4 waves (three workgroups per CU), 128-row tiles of 4
waves (two per CU), 128- and 256-row tiles of 8 waves (one per CU).  The
library picks one by M; the launch settings ARCHEAD_LAUNCH_TILE_WAVES /
ARCHEAD_LAUNCH_TILE_ROWS force each here.

Each layout runs the same cases against the oracle: logits (fp32, a row
stride wider than the row, nothing written past V), CE, the fused argmax and
bf16 logits, at token counts that leave partial tiles (1, 17, 64, 65, 130,
300), on a head whose vocabulary leaves a partial last tile and whose ranks
are not multiples of 16, with fp16 and 8-bit scales; and the tiles' results
agree with each other to the fp32 rounding of their shared arithmetic
(bit for bit: every layout runs the same per-element chain).
"""
from __future__ import annotations


import numpy as np
import pytest

from oracle import head as ohead
from synth import make_head, make_x
from tests.gpu_util import (assert_bf16_output, assert_ce_close, assert_logits_close, say,
                            torch_x)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

LAYOUTS = [("64x4", (4, 64)), ("128x4", (4, 128)), ("8-wave", (8, 0))]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield
    torch.cuda.synchronize()


def _set(ph, layout):
    from paper_2608_02703_amd import archead as ab
    waves, rows = layout
    ph.set_launch(ab.LAUNCH_TILE_WAVES, waves)
    ph.set_launch(ab.LAUNCH_TILE_ROWS, rows)
    assert (ph.get_launch(ab.LAUNCH_TILE_WAVES), ph.get_launch(ab.LAUNCH_TILE_ROWS)) == layout


@pytest.mark.parametrize("scales", ["f16", "u8"])
def test_tile_layouts_match_oracle(scales):
    from paper_2608_02703_amd import PackedHead
    V, d = 1000, 512
    h = make_head("tiny", V=V, d=d, g=64, rc=40, rr=12, scales=scales)
    ph = PackedHead.from_arrays(h)
    ph.force_path("tiled")
    x_all = make_x("tiny", 300, d=d)
    ref_all = ohead.logits(h, x_all)
    got = {}
    try:
        for name, layout in LAYOUTS:
            _set(ph, layout)
            for M in (1, 17, 64, 65, 130, 300):
                say(f"tile layout {name} {scales}: M={M}")
                x, ref = x_all[:M], ref_all[:M]
                out = torch.full((M, V + 5), 3.0, device="cuda")
                ph.logits(torch_x(x), out=out[:, :V])
                torch.cuda.synchronize()
                o = out.cpu().numpy()
                assert (o[:, V:] == 3.0).all(), "wrote past the row"
                lg = o[:, :V]
                assert_logits_close(lg, ref, what=f"{name} M={M}")
                got[(name, M)] = lg
                y = (np.arange(M) * 13 % V).astype(np.int64)
                ce, _ = ph.logits_ce(torch_x(x), torch.from_numpy(y).cuda())
                idx, _ = ph.logits_argmax(torch_x(x))
                torch.cuda.synchronize()
                assert_ce_close(ce.cpu().numpy(), ohead.cross_entropy(ref, y),
                                what=f"{name} M={M} CE")
                assert np.array_equal(idx.cpu().numpy(), np.argmax(lg, axis=1)), \
                    f"{name} M={M}: argmax differs from the first-index argmax of the logits"
                bits = ph.logits(torch_x(x), out_dtype=torch.bfloat16)
                torch.cuda.synchronize()
                bits = bits.view(torch.int16).cpu().numpy().view(np.uint16)
                assert_bf16_output(bits, lg, ref, f"{name} M={M} bf16")
    finally:
        ph.close()
    for M in (1, 17, 64, 65, 130, 300):
        base = got[("64x4", M)]
        for name, _ in LAYOUTS[1:]:
            assert np.array_equal(got[(name, M)].view(np.uint32), base.view(np.uint32)), \
                f"layout {name} differs from 64x4 at M={M}"
