"""Smoke test of the operator comparison harness (WBMM forward against
depthwise convolution, the paper's operator benchmark): one small
configuration runs and reports every method with a finite, positive time.
The harness is context for the paper's comparison, not part of the
operator; its numbers are not checked against anything."""
import math

import pytest

from paper_2607_02097_amd import compare_dw


@pytest.mark.gpu
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_compare_dw_runs(dtype):
    rows = compare_dw.run(dtype, batch=2, maps=[14], channels=8)
    methods = [r["method"] for r in rows]
    assert methods == ["DW-Std 5x5", "DW-Std 13x13", "DW-Std 27x27", "WBMM 7x7", "WBMM 14x14"]
    for r in rows:
        assert r["map"] == 14 and r["batch"] == 2 and r["channels"] == 8 and r["dtype"] == dtype
        assert math.isfinite(r["ms"]) and r["ms"] > 0
        assert math.isfinite(r["kfps"]) and r["kfps"] > 0
        assert r["launch"] in ("graph", "eager")
