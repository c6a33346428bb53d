"""C-ABI contract checks that need no GPU: the library loads, exports every
function include/osoftmax.h declares, and rejects invalid arguments on the
host before touching the device (fake, never dereferenced pointers)."""
import ctypes
import os
import re

import pytest

import paper_1805_02867_amd as osm

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "osoftmax.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return re.findall(r"OSM_API\s+[\w\s\*]+?\b(\w+)\s*\(", text)


def test_header_declares_the_boundary():
    names = declared_functions()
    for want in ("softmax_fwd", "softmax_fwd_ex", "softmax_topk", "softmax_topk_dt",
                 "softmax_topk_ex", "softmax_topk_algo", "topk_fwd", "proj_fwd",
                 "proj_softmax_topk", "osm_plan", "osm_topk_plan", "osm_status_string",
                 "osm_ref_stream", "osm_stream_release"):
        assert want in names


def test_every_declared_symbol_is_exported():
    lib = ctypes.CDLL(osm.LIB_PATH)
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_enum_values_match_header():
    text = open(HEADER).read()
    for name, val in (("OSM_F32", osm.F32), ("OSM_BF16", osm.BF16), ("OSM_NAIVE", osm.NAIVE),
                      ("OSM_SAFE", osm.SAFE), ("OSM_ONLINE", osm.ONLINE), ("OSM_OK", osm.OK),
                      ("OSM_EINVAL", osm.EINVAL), ("OSM_EHIP", osm.EHIP),
                      ("OSM_ENOMEM", osm.ENOMEM), ("OSM_KERNEL_ROWS", osm.KERNEL_ROWS),
                      ("OSM_KERNEL_SPLIT", osm.KERNEL_SPLIT),
                      ("OSM_TOPK_ONLINE_FUSED", osm.TOPK_ONLINE_FUSED),
                      ("OSM_TOPK_SAFE_FUSED", osm.TOPK_SAFE_FUSED),
                      ("OSM_TOPK_SAFE_UNFUSED", osm.TOPK_SAFE_UNFUSED),
                      ("OSM_TOPK_ONLINE_UNFUSED", osm.TOPK_ONLINE_UNFUSED),
                      ("OSM_TOPK_VALUES", osm.TOPK_VALUES)):
        assert re.search(rf"\b{name}\s*=\s*{val}\b", text), name
    assert re.search(rf"#define OSM_TOPK_KMAX {osm.TOPK_KMAX}\b", text)


def test_status_strings():
    for s in range(5):
        assert osm.status_string(s)
    assert osm.status_string(99) == "unknown status"


# Fake device addresses: the validation below must reject these calls before
# any HIP call, so they are never dereferenced.
X, Y = 0x10000000, 0x20000000


@pytest.mark.parametrize("args", [
    (X, Y, -1, 10, 0, 2),          # N < 0
    (X, Y, 4, 0, 0, 2),            # V < 1
    (X, Y, 4, 1 << 31, 0, 2),      # V too large
    (X, Y, 1 << 31, 4, 0, 2),      # N too large
    (X, Y, 4, 10, 2, 2),           # unknown dtype
    (X, Y, 4, 10, 0, 4),           # unknown mode
    (0, Y, 4, 10, 0, 2),           # null x
    (X, 0, 4, 10, 0, 2),           # null y
    (X, X + 8, 4, 10, 0, 2),       # overlap
    (X + 2, Y, 4, 10, 0, 2),       # x not aligned to binary32
    (X, Y + 1, 4, 10, 1, 2),       # y not aligned to bfloat16
])
def test_softmax_fwd_rejects(args):
    assert osm.lib().softmax_fwd(*args, None) == osm.EINVAL


def test_n_zero_is_a_noop():
    assert osm.lib().softmax_fwd(0, 0, 0, 10, 0, 2, None) == osm.OK
    assert osm.lib().softmax_topk(0, 0, 0, 0, 10, 5, None) == osm.OK


@pytest.mark.parametrize("kernel,param", [(7, 0), (1, 3), (1, 2048), (1, 0), (2, 0), (2, -5)])
def test_softmax_fwd_ex_rejects(kernel, param):
    assert osm.lib().softmax_fwd_ex(X, Y, 4, 10, 0, 2, kernel, param, None) == osm.EINVAL


def test_resident_rejects_rows_it_cannot_hold():
    """OSM_RESIDENT holds at most OSM_RESIDENT_MAX_VEC whole 16-byte vectors
    per row; longer rows are refused before any launch."""
    big = osm.RESIDENT_MAX_VEC * 4 + 4          # binary32: one vector too many
    assert osm.lib().softmax_fwd(X, Y, 4, big, 0, osm.RESIDENT, None) == osm.EUNSUPPORTED
    bigb = osm.RESIDENT_MAX_VEC * 8 + 8         # bfloat16
    assert osm.lib().softmax_fwd(X, Y, 4, bigb, 1, osm.RESIDENT, None) == osm.EUNSUPPORTED
    # a forced workgroup size that cannot hold the row
    assert osm.lib().softmax_fwd_ex(X, Y, 4, 32000, 0, osm.RESIDENT, osm.KERNEL_ROWS, 256,
                                    None) == osm.EUNSUPPORTED
    k = ctypes.c_int()
    p = ctypes.c_int64()
    assert osm.lib().osm_plan(4, big, 0, osm.RESIDENT, ctypes.byref(k),
                              ctypes.byref(p)) == osm.EUNSUPPORTED
    assert osm.lib().osm_plan(4, 32000, 0, osm.RESIDENT, ctypes.byref(k), ctypes.byref(p)) == osm.OK
    assert (k.value, p.value) == (osm.KERNEL_ROWS, 512)
    assert osm.lib().osm_plan(4, 128256, 1, osm.RESIDENT, ctypes.byref(k), ctypes.byref(p)) == osm.OK
    assert (k.value, p.value) == (osm.KERNEL_ROWS, 1024)


@pytest.mark.parametrize("kernel,param", [(2, 4), (1, 64), (1, 128), (1, 2048), (7, 0)])
def test_resident_rejects_other_kernels(kernel, param):
    assert osm.lib().softmax_fwd_ex(X, Y, 4, 1000, 0, osm.RESIDENT, kernel, param,
                                    None) == osm.EINVAL


def test_resident_limit_matches_header():
    text = open(HEADER).read()
    assert re.search(rf"#define OSM_RESIDENT_MAX_VEC {osm.RESIDENT_MAX_VEC}\b", text)
    assert re.search(rf"\bOSM_RESIDENT\s*=\s*{osm.RESIDENT}\b", text)


V_, I_ = 0x30000000, 0x40000000


@pytest.mark.parametrize("args", [
    (X, V_, I_, 4, 10, 0),          # K < 1
    (X, V_, I_, 4, 10, 11),         # K > V
    (X, V_, I_, 4, 100, 65),        # K > KMAX
    (0, V_, I_, 4, 10, 5),          # null x
    (X, 0, I_, 4, 10, 5),           # null vals
    (X, V_, 0, 4, 10, 5),           # null idx
    (X, X + 16, I_, 4, 10, 5),      # vals overlaps x
    (X, V_, V_ + 8, 4, 10, 5),      # idx overlaps vals
    (X, V_ + 2, I_, 4, 10, 5),      # misaligned vals
])
def test_softmax_topk_rejects(args):
    assert osm.lib().softmax_topk(*args, None) == osm.EINVAL


@pytest.mark.parametrize("kernel,param", [(2, 0), (2, -3), (2, 1 << 31), (1, 32), (1, 512),
                                          (1, 0), (5, 64)])
def test_softmax_topk_ex_rejects(kernel, param):
    assert osm.lib().softmax_topk_ex(X, V_, I_, 4, 10, 5, 0, kernel, param, None) == osm.EINVAL


Y_ = 0x50000000


@pytest.mark.parametrize("args", [
    (X, Y_, V_, I_, 4, 10, 5, 0, 5, 0, 0),     # unknown algo
    (X, Y_, V_, I_, 4, 10, 5, 0, -1, 0, 0),    # unknown algo
    (X, 0, V_, I_, 4, 10, 5, 0, 2, 0, 0),      # safe unfused without y
    (X, 0, V_, I_, 4, 10, 5, 0, 3, 0, 0),      # online unfused without y
    (X, X + 8, V_, I_, 4, 10, 5, 0, 2, 0, 0),  # y overlaps x
    (X, V_, V_, I_, 4, 10, 5, 0, 3, 0, 0),     # y overlaps vals
    (X, Y_ + 2, V_, I_, 4, 10, 5, 0, 2, 0, 0), # y misaligned
    (X, 0, V_, I_, 4, 10, 5, 0, 1, 1, 128),    # two-wavefront shape: Alg. 4 only
    (X, 0, V_, I_, 4, 10, 5, 0, 4, 1, 128),
    (X, 0, V_, I_, 4, 10, 5, 0, 1, 2, 0),      # split with no chunk
    (X, 0, V_, I_, 4, 10, 11, 0, 1, 0, 0),     # K > V
])
def test_softmax_topk_algo_rejects(args):
    assert osm.lib().softmax_topk_algo(*args, None) == osm.EINVAL


@pytest.mark.parametrize("args", [
    (X, V_, I_, 4, 10, 11, 0),     # K > V
    (X, V_, I_, 4, 10, 0, 0),      # K < 1
    (0, V_, I_, 4, 10, 5, 0),      # null x
    (X, V_, I_, 4, 10, 5, 3),      # unknown dtype
    (X, X + 4, I_, 4, 10, 5, 0),   # vals overlaps x
])
def test_topk_fwd_rejects(args):
    assert osm.lib().topk_fwd(*args, None) == osm.EINVAL


H_, W_, O_ = 0x60000000, 0x70000000, 0x80000000


@pytest.mark.parametrize("args", [
    (H_, W_, O_, -1, 64, 100),           # N < 0
    (H_, W_, O_, 4, 0, 100),             # H < 8
    (H_, W_, O_, 4, 60, 100),            # H not a multiple of 8
    (H_, W_, O_, 4, (1 << 20) + 8, 100), # H above 2^20 (32-bit load offsets in a tile)
    (H_, W_, O_, 4, 64, 0),              # V < 1
    (H_, W_, O_, 65535 * 128 + 1, 64, 10),  # N above the grid limit
    (H_ + 2, W_, O_, 4, 64, 100),        # h not 16-byte aligned
    (H_, W_ + 8, O_, 4, 64, 100),        # w not 16-byte aligned
    (0, W_, O_, 4, 64, 100),             # null h
    (H_, W_, 0, 4, 64, 100),             # null output
    (H_, W_, H_ + 16, 4, 64, 100),       # output overlaps h
])
def test_proj_fwd_rejects(args):
    assert osm.lib().proj_fwd(*args, None) == osm.EINVAL


@pytest.mark.parametrize("args", [
    (H_, W_, V_, I_, 4, 64, 100, 0),     # K < 1
    (H_, W_, V_, I_, 4, 64, 100, 17),    # K > OSM_PROJ_KMAX
    (H_, W_, V_, I_, 4, 64, 10, 11),     # K > V
    (H_, W_, V_, V_ + 4, 4, 64, 100, 5), # idx overlaps vals
    (H_, W_, W_, I_, 4, 64, 100, 5),     # vals overlaps w
    (H_, W_, 0, I_, 4, 64, 100, 5),      # null vals
    (H_, W_, V_, I_, 4, 66, 100, 5),     # H not a multiple of 8
])
def test_proj_softmax_topk_rejects(args):
    assert osm.lib().proj_softmax_topk(*args, None) == osm.EINVAL


def test_proj_accepts_largest_h_without_launch():
    """H = 2^20 passes the checks; N = 0 then returns OSM_OK without a launch."""
    assert osm.lib().proj_fwd(H_, W_, O_, 0, 1 << 20, 100, None) == osm.OK
    assert osm.lib().proj_softmax_topk(H_, W_, V_, I_, 0, 1 << 20, 100, 5, None) == osm.OK


def test_proj_kmax_matches_header():
    assert re.search(rf"#define OSM_PROJ_KMAX {osm.PROJ_KMAX}\b", open(HEADER).read())


def test_softmax_topk_dt_rejects_unknown_dtype():
    assert osm.lib().softmax_topk_dt(X, V_, I_, 4, 10, 5, 7, None) == osm.EINVAL


def test_plan_rejects_bad_shapes():
    k = ctypes.c_int()
    p = ctypes.c_int64()
    assert osm.lib().osm_plan(4, 0, 0, 2, ctypes.byref(k), ctypes.byref(p)) == osm.EINVAL
    assert osm.lib().osm_plan(4, 10, 5, 2, ctypes.byref(k), ctypes.byref(p)) == osm.EINVAL
    assert osm.lib().osm_plan(4, 10, 0, 9, ctypes.byref(k), ctypes.byref(p)) == osm.EINVAL
    assert osm.lib().osm_plan(4, 10, 0, 4, ctypes.byref(k), ctypes.byref(p)) == osm.EINVAL
    assert osm.lib().osm_plan(4, 10, 0, 2, None, ctypes.byref(p)) == osm.EINVAL


def test_topk_plan_rejects_bad_arguments():
    k = ctypes.c_int()
    p = ctypes.c_int64()
    assert osm.lib().osm_topk_plan(4, 0, 0, 5, ctypes.byref(k), ctypes.byref(p)) == osm.EINVAL
    assert osm.lib().osm_topk_plan(4, 10, 0, 11, ctypes.byref(k), ctypes.byref(p)) == osm.EINVAL
    assert osm.lib().osm_topk_plan(4, 100, 0, 65, ctypes.byref(k), ctypes.byref(p)) == osm.EINVAL
    assert osm.lib().osm_topk_plan(4, 10, 0, 5, None, ctypes.byref(p)) == osm.EINVAL


def test_python_binding_refuses_cpu_tensors():
    import torch
    with pytest.raises(ValueError):
        osm.softmax_fwd(torch.zeros(2, 3))
    with pytest.raises(ValueError):
        osm.softmax_topk(torch.zeros(2, 3), 1)
    with pytest.raises(ValueError):
        osm.topk(torch.zeros(2, 3), 1)


@pytest.mark.parametrize("args", [
    (2, H_, W_, 1024),        # unknown op
    (0, H_, W_, -16),         # negative size
    (0, H_, W_, 1000),        # not a multiple of 16
    (0, 0, W_, 1024),         # null x
    (1, H_, 0, 1024),         # null y
    (1, H_ + 4, W_, 1024),    # x not 16-byte aligned
    (1, H_, H_ + 512, 1024),  # copy onto an overlapping y
])
def test_ref_stream_rejects(args):
    assert osm.lib().osm_ref_stream(*args, None) == osm.EINVAL


def test_ref_stream_empty_is_ok_without_launch():
    assert osm.lib().osm_ref_stream(1, H_, W_, 0, None) == osm.OK
