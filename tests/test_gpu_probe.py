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


def test_lds_probe_contiguous_reads_at_full_rate_and_chosen_strides_conflict_free(gpu_lib):
    """The LDS probe: contiguous 16-byte reads cost 4 clocks per CU (256
    bytes per clock); every row stride the kernels use for a pattern costs no
    more than that pattern's best stride among the alternatives, and an
    unpadded 256-byte row (all rows on the same banks) costs several times
    more."""
    import paper_2608_01563_amd as mg
    lin = mg.mg_lds_probe(5, 256, iters=2000)
    say("lds probe: contiguous %.2f clocks" % lin)
    assert 3.0 < lin < 5.0, lin
    # (pattern, stride a kernel uses, alternatives)
    cases = [(0, 288, (272, 304, 320)),   # 16-key dK/dV operand rows (bf16, d = 128)
             (3, 288, (272, 304, 320)),   # its transpose reads
             (2, 304, (272, 288, 320)),   # 32x32x16 operand rows (forward K, dQ K and V)
             (4, 320, (272, 288, 304))]   # forward V transpose reads
    for pattern, used, others in cases:
        t_used = mg.mg_lds_probe(pattern, used, iters=2000)
        t_best = min(mg.mg_lds_probe(pattern, rb, iters=2000) for rb in others)
        say("  pattern %d: stride %d %.2f clocks, best alternative %.2f" % (pattern, used, t_used,
                                                                           t_best))
        assert t_used <= t_best * 1.05, (pattern, used, t_used, t_best)
    assert mg.mg_lds_probe(0, 256, iters=2000) > 3 * lin
