"""The sustained-MFMA probe behind the roofline's measured peak: it must
report a throughput between a third of the published dense peak and the
published peak itself (a figure above it would mean uncounted or dropped
work), for each matrix type."""
import pytest

from gpu_util import say

pytestmark = pytest.mark.gpu

PUBLISHED = {"f32": 157.3, "bf16": 2516.6, "f16": 2516.6}   # MI355X dense, TFLOP/s


@pytest.mark.parametrize("kind", ["f32", "bf16", "f16"])
def test_mfma_probe_in_range(gpu_lib, kind):
    import paper_2608_01563_amd as mg
    tf = mg.mg_mfma_peak(kind, iters=4000)
    say("mfma probe %s: %.1f TFLOP/s" % (kind, tf))
    assert PUBLISHED[kind] / 3 < tf <= PUBLISHED[kind] * 1.02, tf


def test_mfma_probe_argument_errors(gpu_lib):
    import paper_2608_01563_amd as mg
    with pytest.raises(mg.MgError):
        mg.mg_mfma_peak("f32", iters=0)
