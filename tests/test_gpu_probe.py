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
    bytes per clock); every row stride a kernel uses for a pattern costs no
    more than that pattern's best stride among the alternatives, and an
    unpadded 256-byte row (all rows on the same banks) costs several times
    more."""
    import paper_2608_01563_amd as mg
    lin = mg.mg_lds_probe(5, 256, iters=2000)
    say("lds probe: contiguous %.2f clocks" % lin)
    assert 3.0 < lin < 5.0, lin
    # (pattern, stride a kernel uses, alternatives)
    cases = [(2, 304, (272, 288, 320)),   # 32x32x16 operand rows (accelerated forward K)
             (4, 320, (272, 288, 304)),   # its V transpose reads
             (1, 272, (256, 288, 304))]   # f32 16x16x4 operand groups (fused backward)
    for pattern, used, others in cases:
        t_used = mg.mg_lds_probe(pattern, used, iters=2000)
        t_best = min(mg.mg_lds_probe(pattern, rb, iters=2000) for rb in others)
        say("  pattern %d: stride %d %.2f clocks, best alternative %.2f" % (pattern, used, t_used,
                                                                           t_best))
        assert t_used <= t_best * 1.05, (pattern, used, t_used, t_best)
    assert mg.mg_lds_probe(0, 256, iters=2000) > 3 * lin


def test_lds_probe_block_layouts_at_the_minimum(gpu_lib):
    """The bf16 kernels' swizzled column-block tiles: their 16-byte reads
    cost what contiguous reads cost (no bank conflicts), their transpose
    reads cost no more than the cheapest padded stride achieves for the same
    shape, and without the swizzle the 16-byte reads cost at least half as
    much again."""
    import paper_2608_01563_amd as mg
    lin = mg.mg_lds_probe(5, 256, iters=2000)
    tr_best = min(mg.mg_lds_probe(3, 288, iters=2000), mg.mg_lds_probe(4, 320, iters=2000))
    for pattern, rb, kind in ((7, 64, "b128"), (8, 64, "tr"), (9, 64, "b128"),
                              (10, 64, "tr"), (11, 128, "tr")):
        t = mg.mg_lds_probe(pattern, rb, iters=2000)
        plain = mg.mg_lds_probe(pattern + 5, rb, iters=2000)
        say("  block pattern %d: %.2f clocks swizzled, %.2f unswizzled" % (pattern, t, plain))
        if kind == "b128":
            assert t <= lin * 1.05, (pattern, t, lin)
            assert plain >= 1.5 * t, (pattern, plain, t)
        else:
            assert t <= tr_best * 1.05, (pattern, t, tr_best)
    with pytest.raises(mg.MgError):
        mg.mg_lds_probe(7, 128)            # pattern 7 reads 64-byte block rows


def test_lds_probe_f32_forward_tiles_at_the_best_padding(gpu_lib):
    """The strict f32 forward's chunk-permuted K and V tiles (d = 64): each
    read costs no more than the cheapest padded stride achieves for the same
    read shape, and the 16x16x4 operand groups cost several times more on
    unpermuted 256-byte rows."""
    import paper_2608_01563_amd as mg
    for pattern, shape in ((17, 1), (18, 6)):
        t = mg.mg_lds_probe(pattern, 256, iters=2000)
        best = min(mg.mg_lds_probe(shape, rb, iters=2000) for rb in (272, 288, 304, 336))
        say("  f32 forward pattern %d: %.2f clocks, best padded stride %.2f" % (pattern, t, best))
        assert t <= best * 1.05, (pattern, t, best)
    assert mg.mg_lds_probe(1, 256, iters=2000) > 2 * mg.mg_lds_probe(17, 256, iters=2000)
