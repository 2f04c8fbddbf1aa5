"""How far two correct float32 accumulation orders of one bf16 model drift apart
(CPU, slow): the measurement the GPU's end-to-end bf16 bar rests on.

The oracle's "bf16" mode (float32 products) and "bf16_f64acc" mode (float64
products, the same bf16 rounding points) run the LLaDA-8B-shaped model on the
workload's first input for 1, 2, 4 and 8 layers; the block's logits and
confidences (Box 1) are compared at each depth.  The committed table
tests/golden/bf16_drift_llada.json (written by make_drift_table.py, depths to
32) must reproduce within a factor of two (BLAS thread counts change which
values flip), the logit spread must grow with depth, and the confidence spread
must stay below 2e-2.
"""
import json
import os
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.join(HERE, "golden"))

pytestmark = pytest.mark.slow


def test_bf16_accumulation_drift_by_depth():
    from make_drift_table import OUT, drift
    table = {r["depth"]: r for r in json.load(open(OUT))["rows"]}
    got = drift([1, 2, 4, 8], log=print)
    prev = 0.0
    for r in got:
        ref = table[r["depth"]]
        for key in ("logit_max_abs_diff", "conf_max_abs_diff"):
            assert 0.5 * ref[key] <= r[key] <= 2.0 * ref[key], (r["depth"], key, r[key], ref[key])
        assert r["logit_max_abs_diff"] > prev
        prev = r["logit_max_abs_diff"]
        assert r["conf_max_abs_diff"] < 2e-2
    # even one layer drifts past the flat 2e-2 logit bar: the bar must follow the table
    assert got[0]["logit_max_abs_diff"] > 2e-2
