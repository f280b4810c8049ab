"""The C ABI library loads and exports every entry point of include/saef.h,
and its host-side argument checks work without a GPU."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "saef.h")


def header_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^int\s+(saef_\w+)\s*\(", text, flags=re.M)))


@pytest.fixture(scope="module")
def saef():
    from paper_2008_05823_amd import saef as mod
    return mod


def test_header_declares_the_entry_points():
    names = header_functions()
    for required in ("saef_compress", "saef_aggregate", "saef_step_ahead",
                     "saef_error_average", "saef_round", "saef_layout_create",
                     "saef_layout_destroy", "saef_status", "saef_materialize"):
        assert required in names


def test_library_exports_every_declared_symbol(saef):
    lib = ctypes.CDLL(saef.LIB_PATH)
    for name in header_functions():
        assert hasattr(lib, name), f"{name} declared in saef.h but not exported"
    assert sorted(saef.EXPORTS) == header_functions()


def test_layout_create_rejects_bad_layouts_on_host(saef):
    lib = saef.raw_library()
    h = ctypes.c_void_p()

    def create(off, n, d_pad, k_max=2):
        o = (ctypes.c_int64 * len(off))(*off)
        s = (ctypes.c_int64 * len(n))(*n)
        return lib.saef_layout_create(o, s, len(off), d_pad, k_max, ctypes.byref(h))

    assert create([32], [10], 64) == saef.EINVAL            # offset not 64-aligned
    assert create([0, 64], [100, 10], 192) == saef.EINVAL   # overlap
    assert create([0], [0], 64) == saef.EINVAL              # empty tensor
    assert create([0], [65], 64) == saef.EINVAL             # past d_pad
    assert create([0], [10], 64, k_max=0) == saef.EINVAL    # no workers
    assert create([0], [1 << 29], 1 << 29) == saef.EINVAL   # above 2^28 elements
    assert h.value is None


def test_null_layout_is_rejected(saef):
    lib = saef.raw_library()
    assert lib.saef_layout_destroy(None) == saef.EINVAL
    assert lib.saef_status(None, None) == saef.EINVAL
    assert lib.saef_compress(None, 1, ctypes.c_float(0.1), None, None, None, None,
                             None) == saef.EINVAL
    assert lib.saef_round(None, 0, 0, 1, ctypes.c_float(0.1), 1, *([None] * 10)) == saef.EINVAL


def test_profile_calls_reject_bad_arguments_on_host(saef):
    lib = saef.raw_library()
    counts = (ctypes.c_int32 * 7)()
    ms = (ctypes.c_double * 7)()
    assert lib.saef_profile_enable(None, 4, 1, 1) == saef.EINVAL   # no layout
    assert lib.saef_profile_read(None, counts, ms) == saef.EINVAL


def test_topk_calls_reject_null_plans_on_host(saef):
    lib = saef.raw_library()
    assert lib.saef_topk_materialize(None, 1, None, None, None) == saef.EINVAL
    assert lib.saef_topk_round_begin(None, 0, 0, 1, 1, 1, *([None] * 7)) == saef.EINVAL
    assert lib.saef_topk_round_end(None, 0, 0, 1, ctypes.c_float(0.1), ctypes.c_float(0.0), 1,
                                   *([None] * 12)) == saef.EINVAL


@pytest.mark.gpu
def test_alignment_rule_on_device(saef):
    """Buffers must be aligned to their element type, no more: a float buffer
    4 bytes past a 256-byte boundary is accepted, one 2 bytes past is
    SAEF_EINVAL (nothing enqueued); sign words need 8 bytes."""
    import torch
    from paper_2008_05823_amd import workloads as W
    w = W.custom([100, 70], K=2)
    off, n, d_pad = w.layout()
    lay = saef.Layout(off, n, d_pad, 2)
    lib = saef.raw_library()
    f32 = dict(dtype=torch.float32, device="cuda")
    g = torch.zeros(2 * d_pad + 8, **f32)
    e = torch.zeros(2 * d_pad + 8, **f32)
    words = torch.zeros(2 * (d_pad // 64) + 2, dtype=torch.int64, device="cuda")
    scales = torch.zeros(2 * w.L + 4, **f32)
    s = torch.cuda.current_stream().cuda_stream

    def compress(g_ptr, e_ptr, w_ptr):
        return lib.saef_compress(lay.handle, 2, ctypes.c_float(0.1), g_ptr, e_ptr, w_ptr,
                                 scales.data_ptr(), s)

    base_w = words.data_ptr()
    assert compress(g.data_ptr() + 4, e.data_ptr() + 4, base_w) == saef.OK
    assert compress(g.data_ptr() + 2, e.data_ptr(), base_w) == saef.EINVAL
    assert compress(g.data_ptr(), e.data_ptr() + 2, base_w) == saef.EINVAL
    assert compress(g.data_ptr(), e.data_ptr(), base_w + 4) == saef.EINVAL
    assert compress(g.data_ptr(), e.data_ptr(), base_w + 8) == saef.OK
    torch.cuda.synchronize()
    assert saef.saef_status(lay) == saef.OK
    lay.close()
