"""Host-side checks of bench.py's accounting (no GPU): every kernel stage the
library can name in its timing hooks has an algorithmic-work entry, so that
`roofline` and the per-kernel table never meet an unknown kernel."""
import os
import re

import pytest

import bench
from workloads import WORKLOADS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _stages():
    src = open(os.path.join(ROOT, "paper_2608_01563_amd", "csrc", "mg_attn.cpp")).read()
    return sorted(set(re.findall(r'kernel_name\("([a-z_]+)"', src)))


def test_the_library_names_its_stages():
    assert {"attn_fwd", "attn_rowdot", "attn_dkdvq", "attn_dqreduce",
            "attn_bwdreduce"} <= set(_stages())


@pytest.mark.parametrize("wid", sorted(WORKLOADS))
@pytest.mark.parametrize("stage", _stages())
def test_every_stage_has_algorithmic_work(stage, wid):
    w = WORKLOADS[wid]
    suffix = {"strict_f32": "f32", "fast_bf16": "bf16", "accelerated": "accel"}[w.contract]
    pairs = 1000.0
    rows = w.B * w.H * w.L
    amount, unit, bound = bench.kernel_work("%s_%s_d%d" % (stage, suffix, w.d), w, pairs, rows)
    assert amount > 0 and unit in ("flop", "byte") and bound in ("mfma", "hbm")
    # the combined reduction moves at least what the dQ reduction alone moves
    if stage == "attn_bwdreduce":
        dq, _, _ = bench.kernel_work("attn_dqreduce_%s_d%d" % (suffix, w.d), w, pairs, rows)
        assert amount > dq
