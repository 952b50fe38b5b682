"""Host-side checks of the C-ABI library (no GPU needed): it builds, loads,
exports every entry point its header declares, and rejects bad arguments on
the host before anything is enqueued."""
import ctypes
import os
import re
import subprocess

import pytest

import paper_2608_01563_amd as mg
from paper_2608_01563_amd import _binding


def header_functions():
    names = set()
    for path in (mg.HEADER_PATH, mg.CONV_HEADER_PATH):
        with open(path) as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        names.update(re.findall(r"\b(mg_[a-z_0-9]+)\s*\(", text))
    return sorted(names)


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(mg.LIB_PATH):
        pytest.fail("libmg.so is not built; run __graft_entry__.build()")
    return mg.load_library()


def test_header_declares_the_boundary():
    names = header_functions()
    for required in ("mg_attn_fwd", "mg_attn_bwd", "mg_attn_bwd_workspace_bytes",
                     "mg_status_string", "mg_last_error_detail", "mg_conv2d_bwd_data",
                     "mg_conv2d_bwd_filter", "mg_conv2d_bwd_filter_workspace_bytes"):
        assert required in names


def test_every_declared_symbol_is_exported(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", mg.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = {line.split()[-1] for line in out.splitlines() if " T " in line}
    for name in header_functions():
        assert name in exported, name
        assert hasattr(lib, name)


def test_status_strings(lib):
    for code, name in _binding.STATUS_NAMES.items():
        assert mg.mg_status_string(code) == name
    assert mg.mg_status_string(99) == "MG_ERR_UNKNOWN"


def test_workspace_query(lib):
    rows = 8 * 8 * 1024
    # strict f32, d <= 64: D plus one dQ partial per (key tile, query row);
    # key tiles hold 128 keys under a causal mask with >= 512 such tiles, else 64
    assert mg.mg_attn_bwd_workspace_bytes(8, 8, 1024, 64, 1, 0) == rows * 4 + 8 * rows * 64 * 4
    assert mg.mg_attn_bwd_workspace_bytes(8, 8, 1024, 64, 0, 0) == rows * 4 + 16 * rows * 64 * 4
    # bf16, or d = 128: D only
    assert mg.mg_attn_bwd_workspace_bytes(8, 8, 1024, 64, 1, 1) == rows * 4
    assert mg.mg_attn_bwd_workspace_bytes(8, 8, 1024, 128, 1, 0) == rows * 4
    # partials above 1 GiB fall back to the separate dQ kernel (D only)
    assert mg.mg_attn_bwd_workspace_bytes(8, 8, 8192, 64, 0, 0) == 8 * 8 * 8192 * 4
    assert mg.mg_attn_bwd_workspace_bytes(1, 1, 3, 32, 0, 0) == 256 + 3 * 32 * 4
    # causal but too few 128-key tiles: 64-key tiles (B4 H4 L256 -> 4 tiles);
    # 64 workgroups split each key tile's 8 query tiles (a short query side:
    # shares down to 2 tiles) in S = min(16, 8/2) = 4
    assert mg.mg_attn_bwd_workspace_bytes(4, 4, 256, 64, 1, 0) == \
        4096 * 4 + 4 * 4096 * 64 * 4 + 2 * 4 * 16 * 256 * 64 * 4
    assert mg.mg_attn_bwd_workspace_bytes(1, 1, 3, 48, 0, 0) == 0     # unsupported d
    assert mg.mg_attn_bwd_workspace_bytes(0, 1, 3, 32, 0, 0) == 0     # bad size
    assert mg.mg_attn_bwd_workspace_bytes(1, 1, 3, 32, 0, 7) == 0     # bad contract
    # the accelerated contract's backward is the strict one: same workspace
    for args in ((8, 8, 1024, 64, 1), (8, 8, 1024, 64, 0), (8, 8, 1024, 128, 1),
                 (4, 4, 256, 64, 1), (1, 1, 3, 32, 0)):
        assert mg.mg_attn_bwd_workspace_bytes(*args, 2) == mg.mg_attn_bwd_workspace_bytes(*args, 0)


def test_cross_workspace_query(lib):
    # D has one f32 per query row; the fused dQ partials are
    # ceil(Lk / key_rows) * B*H*Lq*d f32, key tiles decided from Lk
    B, H, Lq, Lk, d = 4, 8, 1024, 77, 64
    rows = B * H * Lq
    # 2 key tiles x 32 heads = 64 workgroups: S = min(1024/64, (1024/32)/4) = 8
    assert mg.mg_attn_bwd_cross_workspace_bytes(B, H, Lq, Lk, d, 0, 0) == \
        rows * 4 + 2 * rows * d * 4 + 2 * 8 * B * H * Lk * d * 4
    assert mg.mg_attn_bwd_cross_workspace_bytes(B, H, Lq, Lk, d, 0, 1) == rows * 4
    assert mg.mg_attn_bwd_cross_workspace_bytes(B, H, Lq, Lk, d, 0, 2) == \
        mg.mg_attn_bwd_cross_workspace_bytes(B, H, Lq, Lk, d, 0, 0)
    # 50 action queries onto 66 keys: D rounded up to 256 bytes; two query
    # tiles are too few to split
    assert mg.mg_attn_bwd_cross_workspace_bytes(1, 1, 50, 66, 32, 1, 0) == 256 + 2 * 50 * 32 * 4
    # causal, Lk = 1024 with 8*8 heads -> 512 tiles of 128 keys over Lq = 300 rows
    assert mg.mg_attn_bwd_cross_workspace_bytes(8, 8, 300, 1024, 64, 1, 0) == \
        64 * 300 * 4 + 8 * 64 * 300 * 64 * 4
    # the square entry points are the cross ones with Lq = Lk
    for args in ((8, 8, 1024, 64, 1, 0), (4, 4, 256, 64, 1, 0), (1, 1, 3, 32, 0, 1)):
        B, H, L, d, c, k = args
        assert mg.mg_attn_bwd_workspace_bytes(*args) == \
            mg.mg_attn_bwd_cross_workspace_bytes(B, H, L, L, d, c, k)
    assert mg.mg_attn_bwd_cross_workspace_bytes(1, 1, 3, 0, 32, 0, 0) == 0    # Lk < 1
    assert mg.mg_attn_bwd_cross_workspace_bytes(1, 1, 0, 3, 32, 0, 0) == 0    # Lq < 1


def test_cross_forward_size_checks(lib):
    vp = ctypes.c_void_p
    Q, K, V, O, LSE = (vp(p) for p in GOOD)

    def fwd(Lq, Lk, B=1, H=1, d=64):
        return lib.mg_attn_fwd_cross(Q, K, V, O, LSE, None, B, H, Lq, Lk, d, 1,
                                     ctypes.c_float(0.125), 0, None)
    assert fwd(8, 0) == 1 and fwd(0, 8) == 1
    # the element-count limit applies to the longer of the two lengths
    assert fwd(4, 1 << 22, B=1 << 4, H=1 << 1) == 1
    assert fwd(1 << 22, 4, B=1 << 4, H=1 << 1) == 1
    assert "2^31" in mg.mg_last_error_detail()


def _fwd(lib, ptrs, B=1, H=1, L=8, d=64, scale=0.125, contract=0):
    Q, K, V, O, LSE = ptrs
    vp = ctypes.c_void_p
    return lib.mg_attn_fwd(vp(Q), vp(K), vp(V), vp(O), vp(LSE), None, B, H, L, d, 1,
                           ctypes.c_float(scale), contract, None)


GOOD = [0x1000, 0x2000, 0x3000, 0x4000, 0x5000]   # aligned, never dereferenced


@pytest.mark.parametrize("kwargs,status", [
    (dict(B=0), 1), (dict(H=-1), 1), (dict(L=0), 1), (dict(d=0), 1),
    (dict(d=48), 2), (dict(d=256), 2),
    (dict(scale=float("inf")), 1), (dict(scale=float("nan")), 1),
    (dict(contract=5), 1),
    (dict(B=1 << 12, H=1 << 10, L=1 << 10, d=64), 1),   # B*H*L*d > 2^31-1
])
def test_forward_rejects_bad_sizes_before_any_device_call(lib, kwargs, status):
    assert _fwd(lib, GOOD, **kwargs) == status
    assert mg.mg_last_error_detail() != ""


def test_forward_rejects_null_and_misaligned_pointers(lib):
    for k in range(5):
        ptrs = list(GOOD)
        ptrs[k] = 0
        assert _fwd(lib, ptrs) == 1
        ptrs[k] = GOOD[k] + 4
        assert _fwd(lib, ptrs) == 3


def test_backward_rejects_missing_workspace(lib):
    vp = ctypes.c_void_p
    ptrs = [vp(0x1000 * (k + 1)) for k in range(9)]
    st = lib.mg_attn_bwd(*ptrs, None, 1, 1, 8, 64, 1, ctypes.c_float(0.125), 0,
                         None, 0, None)
    assert st == 4                 # checked before any pointer reaches the runtime
    st = lib.mg_attn_bwd(*ptrs, None, 1, 1, 8, 64, 1, ctypes.c_float(0.125), 9,
                         None, 0, None)
    assert st == 1


def test_host_memory_is_refused(lib):
    bufs = [ctypes.create_string_buffer(4096 + 16) for _ in range(5)]
    ptrs = [(ctypes.addressof(b) + 15) // 16 * 16 for b in bufs]
    assert _fwd(lib, ptrs) == 1
    assert "device" in mg.mg_last_error_detail()


# ---- convolution derivatives (include/mg_conv.h)

def _shape(N=1, H=8, W=8, C=4, K=8, R=3, S=3, sh=1, sw=1, ph=1, pw=1):
    return _binding.ConvShape(N, H, W, C, K, R, S, sh, sw, ph, pw)


def test_conv_workspace_query(lib):
    # ResNet-50's first layer at batch 4: 3 output tiles (64 x 147 of dW) over
    # 4*112*112 positions in 3136 16-deep steps -> min(ceil(1024/3), 3136/16) = 196 splits
    s = _shape(4, 224, 224, 3, 64, 7, 7, 2, 2, 3, 3)
    assert lib.mg_conv2d_bwd_filter_workspace_bytes(ctypes.byref(s), 0) == 196 * 64 * 147 * 4
    # a 3x3 512->512 layer at 7x7: the filter gradient's 8 x 72 = 576 tiles fill
    # the GPU (no workspace); its data gradient has 4 x 8 = 32 tiles over 288
    # steps -> min(32, 288/16) = 18 splits of the 196 x 512 output
    s = _shape(4, 7, 7, 512, 512, 3, 3, 1, 1, 1, 1)
    assert lib.mg_conv2d_bwd_filter_workspace_bytes(ctypes.byref(s), 0) == 0
    assert lib.mg_conv2d_bwd_data_workspace_bytes(ctypes.byref(s), 0) == 18 * 196 * 512 * 4
    # a stride-2 3x3 layer: four parity classes (taps 2x2, 2x1, 1x2, 1x1) of
    # 7x7, 7x7, 7x7, 7x7 pixels at batch 4 -> 4 tiles each x 4 channel tiles
    # = 64 tiles, the longest class sums 4 taps x 256 = 64 steps -> min(16, 4)
    s2 = _shape(4, 14, 14, 256, 256, 3, 3, 2, 2, 1, 1)
    assert lib.mg_conv2d_bwd_data_workspace_bytes(ctypes.byref(s2), 0) == 4 * 4 * 14 * 14 * 256 * 4
    # both at once: the data gradient's partials, 256-byte aligned, then the
    # filter gradient's
    s3 = _shape(4, 14, 14, 256, 256, 3, 3, 1, 1, 1, 1)
    d = lib.mg_conv2d_bwd_data_workspace_bytes(ctypes.byref(s3), 0)
    w = lib.mg_conv2d_bwd_filter_workspace_bytes(ctypes.byref(s3), 0)
    assert d > 0 and w > 0
    assert lib.mg_conv2d_bwd_workspace_bytes(ctypes.byref(s3), 0) == (d + 255) // 256 * 256 + w
    assert lib.mg_conv2d_bwd_workspace_bytes(ctypes.byref(s), 0) == \
        lib.mg_conv2d_bwd_data_workspace_bytes(ctypes.byref(s), 0)     # filter: no split
    # 56x56 at batch 4 with 256 channels: 196 x 4 = 784 tiles, no split
    s = _shape(4, 56, 56, 256, 64, 1, 1, 1, 1, 0, 0)
    assert lib.mg_conv2d_bwd_data_workspace_bytes(ctypes.byref(s), 0) == 0
    # accelerated = strict; bf16, bad sizes and a filter larger than the
    # padded input give 0
    s = _shape(4, 56, 56, 64, 64, 1, 1, 1, 1, 0, 0)
    assert lib.mg_conv2d_bwd_filter_workspace_bytes(ctypes.byref(s), 2) == \
        lib.mg_conv2d_bwd_filter_workspace_bytes(ctypes.byref(s), 0) > 0
    assert lib.mg_conv2d_bwd_filter_workspace_bytes(ctypes.byref(s), 1) == 0
    assert lib.mg_conv2d_bwd_filter_workspace_bytes(ctypes.byref(_shape(C=0)), 0) == 0
    assert lib.mg_conv2d_bwd_filter_workspace_bytes(
        ctypes.byref(_shape(H=2, W=2, R=5, S=5, ph=1, pw=1)), 0) == 0


@pytest.mark.parametrize("kwargs,status", [
    (dict(N=0), 1), (dict(C=-1), 1), (dict(R=0), 1), (dict(sh=0), 1), (dict(pw=-1), 1),
    (dict(H=2, R=5, ph=1), 1),                                   # no output row
    (dict(N=64, H=512, W=512, C=64), 1),                         # X above 2^31-1 bytes
])
def test_conv_rejects_bad_shapes_before_any_device_call(lib, kwargs, status):
    vp = ctypes.c_void_p
    s = _shape(**kwargs)
    assert lib.mg_conv2d_bwd_data(vp(0x1000), vp(0x2000), vp(0x3000), ctypes.byref(s), 0,
                                  None, 0, None) == status
    assert mg.mg_last_error_detail() != ""


def test_conv_contracts_and_pointers(lib):
    vp = ctypes.c_void_p
    s = _shape()
    call = lambda a, b, c, shp, k: lib.mg_conv2d_bwd_data(a, b, c, shp, k, None, 0, None)
    assert call(vp(0x1000), vp(0x2000), vp(0x3000), ctypes.byref(s), 1) == 2   # no bf16
    assert call(vp(0x1000), vp(0x2000), vp(0x3000), ctypes.byref(s), 7) == 1
    assert call(vp(0x1000), None, vp(0x3000), ctypes.byref(s), 0) == 1
    assert call(vp(0x1004), vp(0x2000), vp(0x3000), ctypes.byref(s), 0) == 3
    assert call(vp(0x1000), vp(0x2000), vp(0x3000), None, 0) == 1
    s7 = _shape(4, 7, 7, 512, 512, 3, 3, 1, 1, 1, 1)
    assert call(vp(0x1000), vp(0x2000), vp(0x3000), ctypes.byref(s7), 0) == 4  # workspace
    big = _shape(4, 224, 224, 3, 64, 7, 7, 2, 2, 3, 3)
    assert lib.mg_conv2d_bwd_filter(vp(0x1000), vp(0x2000), vp(0x3000), ctypes.byref(big), 0,
                                    None, 0, None) == 4          # workspace needed


def test_conv_fused_entry_point_checks(lib):
    vp = ctypes.c_void_p
    s = _shape()
    args = [vp(0x1000), vp(0x2000), vp(0x3000), vp(0x4000), vp(0x5000)]
    assert lib.mg_conv2d_bwd(*args, ctypes.byref(s), 1, None, 0, None) == 2
    args[3] = None
    assert lib.mg_conv2d_bwd(*args, ctypes.byref(s), 0, None, 0, None) == 1
    big = _shape(4, 7, 7, 512, 512, 3, 3, 1, 1, 1, 1)
    args[3] = vp(0x4000)
    assert lib.mg_conv2d_bwd(*args, ctypes.byref(big), 0, None, 0, None) == 4


def test_mfma_probe_rejects_bad_arguments_before_any_device_call(lib):
    out = ctypes.c_double(0.0)
    assert lib.mg_mfma_peak(3, 100, ctypes.byref(out), None) == 1
    assert lib.mg_mfma_peak(-1, 100, ctypes.byref(out), None) == 1
    assert lib.mg_mfma_peak(0, 0, ctypes.byref(out), None) == 1
    assert lib.mg_mfma_peak(0, (1 << 24) + 1, ctypes.byref(out), None) == 1
    assert lib.mg_mfma_peak(1, 100, None, None) == 1
    assert mg.mg_last_error_detail() != ""


def test_lds_probe_rejects_bad_arguments_before_any_device_call(lib):
    out = ctypes.c_double(0.0)
    # block-layout patterns (7..16) take their block row only (64, or 128 for 11 and 16)
    for args in ((7, 256, 100), (11, 64, 100), (16, 64, 100), (17, 64, 100), (18, 128, 100), (19, 256, 100), (-1, 256, 100),
                 (0, 8, 100), (0, 488, 100), (0, 264, 100), (0, 256, 0),
                 (0, 256, (1 << 20) + 1)):
        assert lib.mg_lds_probe(*args, ctypes.byref(out), None) == 1, args
    assert lib.mg_lds_probe(0, 256, 100, None, None) == 1
    assert mg.mg_last_error_detail() != ""


def test_error_detail_is_per_thread(lib):
    """mg_last_error_detail describes the calling thread's last call only."""
    import threading
    seen = {}

    def fresh():
        seen["fresh"] = mg.mg_last_error_detail()

    def failing():
        assert _fwd(lib, GOOD, d=48) == 2
        seen["own"] = mg.mg_last_error_detail()

    assert _fwd(lib, GOOD, B=0) == 1
    mine = mg.mg_last_error_detail()
    for target in (fresh, failing):
        t = threading.Thread(target=target)
        t.start()
        t.join()
    assert seen["fresh"] == ""
    assert seen["own"] != "" and seen["own"] != mine
    assert mg.mg_last_error_detail() == mine   # untouched by the other threads
