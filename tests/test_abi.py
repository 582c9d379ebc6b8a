"""The C ABI library loads, exports what include/eb.h declares, and rejects bad
arguments before touching a device (CPU only: no compute calls)."""
import ctypes
import os
import re
import subprocess

import pytest

from paper_2609_30656_amd import eb

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "eb.h")


def _declared():
    text = open(HEADER).read()
    return set(re.findall(r"^\s*(?:eb_status|const char \*)\s*(eb_\w+)\s*\(", text, re.M))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(eb.LIB_PATH):
        pytest.skip("libeb.so not built")
    return eb.load_library()


def test_exports_match_header(lib):
    declared = _declared()
    assert declared == set(eb.EXPORTED)
    for name in declared:
        assert hasattr(lib, name)
    nm = subprocess.run(["nm", "-D", "--defined-only", eb.LIB_PATH], capture_output=True, text=True, check=True)
    exported = {ln.split()[-1] for ln in nm.stdout.splitlines() if " T " in ln}
    assert exported == declared  # nothing else leaks out of the library


def test_noalloc_workspace_size_matches_header():
    m = re.search(r"^#define EB_NOALLOC_SCRATCH_BYTES (\d+)", open(HEADER).read(), re.M)
    assert m and int(m.group(1)) == eb.EB_NOALLOC_SCRATCH_BYTES == 128 << 20


def test_noalloc_rejects_null_handle(lib):
    none = eb._as_tensor(None)
    assert lib.eb_backward_update_noalloc(None, none, none, none, 0, none, 0, ctypes.c_float(0.1),
                                          ctypes.c_float(0.0), none) == eb.EB_ERR_INVALID_ARG


def test_status_strings(lib):
    codes = [eb.EB_OK, eb.EB_ERR_INVALID_ARG, eb.EB_ERR_DTYPE, eb.EB_ERR_SHAPE, eb.EB_ERR_UNSUPPORTED,
             eb.EB_ERR_INDEX_OOB, eb.EB_ERR_OFFSETS, eb.EB_ERR_OOM, eb.EB_ERR_HIP]
    msgs = [eb.eb_status_string(c) for c in codes]
    assert len(set(msgs)) == len(msgs)
    assert eb.eb_status_string(12345) == "unknown status"


_buf = ctypes.create_string_buffer(4096 + 64)
_ALIGNED = (ctypes.addressof(_buf) + 63) // 64 * 64  # host address: never dereferenced here


def _create(lib, descs, n=None, out=True):
    arr = (eb.eb_table_desc * max(len(descs), 1))(*descs)
    h = ctypes.c_void_p(0xDEAD)
    st = lib.eb_create_tables(arr if descs else None, len(descs) if n is None else n, None,
                              ctypes.byref(h) if out else None)
    return st, h.value


def _desc(data=_ALIGNED, rows=10, dim=16, dtype=eb.EB_F32, stride=None):
    if stride is None:
        stride = dim * {eb.EB_F32: 4, eb.EB_F16: 2, eb.EB_INT8_ROWWISE: 1, eb.EB_INT8_ROWWISE_SPLIT: 1}.get(
            dtype, 4) + (4 if dtype == eb.EB_INT8_ROWWISE else 0)
    return eb.eb_table_desc(data, rows, dim, dtype, stride)


@pytest.mark.parametrize("desc, expect", [
    (dict(data=None), eb.EB_ERR_INVALID_ARG),
    (dict(rows=0), eb.EB_ERR_INVALID_ARG),
    (dict(rows=1 << 31), eb.EB_ERR_INVALID_ARG),
    (dict(dim=0), eb.EB_ERR_INVALID_ARG),
    (dict(dim=16384), eb.EB_ERR_INVALID_ARG),
    (dict(dtype=7), eb.EB_ERR_DTYPE),
    (dict(dim=6), eb.EB_ERR_UNSUPPORTED),                                   # fp32 needs dim % 4
    (dict(dim=12, dtype=eb.EB_F16), eb.EB_ERR_UNSUPPORTED),                 # fp16 needs dim % 8
    (dict(dim=24, dtype=eb.EB_INT8_ROWWISE), eb.EB_ERR_UNSUPPORTED),        # int8 needs dim % 16
    (dict(stride=32), eb.EB_ERR_INVALID_ARG),                               # shorter than a row
    (dict(stride=72), eb.EB_ERR_UNSUPPORTED),                               # fp32 stride % 16
    (dict(data=_ALIGNED + 4), eb.EB_ERR_UNSUPPORTED),                       # fp32 rows 16-B aligned
    (dict(dim=128, dtype=eb.EB_INT8_ROWWISE, stride=130), eb.EB_ERR_INVALID_ARG),
    (dict(dim=128, dtype=eb.EB_INT8_ROWWISE, stride=134), eb.EB_ERR_UNSUPPORTED),
    (dict(dim=128, dtype=eb.EB_INT8_ROWWISE, data=_ALIGNED + 2), eb.EB_ERR_UNSUPPORTED),
    (dict(dim=24, dtype=eb.EB_INT8_ROWWISE_SPLIT), eb.EB_ERR_UNSUPPORTED),  # split int8: dim % 16
    (dict(dim=128, dtype=eb.EB_INT8_ROWWISE_SPLIT, stride=112), eb.EB_ERR_INVALID_ARG),  # shorter than the codes
    (dict(dim=128, dtype=eb.EB_INT8_ROWWISE_SPLIT, stride=132), eb.EB_ERR_UNSUPPORTED),  # stride % 16
    (dict(dim=128, dtype=eb.EB_INT8_ROWWISE_SPLIT, data=_ALIGNED + 4), eb.EB_ERR_UNSUPPORTED),  # 16-B aligned
    (dict(dtype=4), eb.EB_ERR_DTYPE),
])
def test_create_rejects_bad_descriptors(lib, desc, expect):
    st, h = _create(lib, [_desc(), _desc(**desc)])
    assert st == expect
    assert h is None  # *out is cleared on error


def test_create_rejects_bad_calls(lib):
    assert _create(lib, [_desc()], out=False)[0] == eb.EB_ERR_INVALID_ARG
    assert _create(lib, [], n=1)[0] == eb.EB_ERR_INVALID_ARG
    assert _create(lib, [_desc()], n=0)[0] == eb.EB_ERR_INVALID_ARG
    assert _create(lib, [_desc()], n=-3)[0] == eb.EB_ERR_INVALID_ARG


def test_forward_and_destroy_on_null_handle(lib):
    t = eb.eb_tensor(None, 0, eb.EB_I64)
    o = eb.eb_tensor(None, 0, eb.EB_T_F32)
    assert lib.eb_forward(None, t, t, o, eb.EB_POOL_SUM, o) == eb.EB_ERR_INVALID_ARG
    assert lib.eb_destroy(None) == eb.EB_OK


def test_valid_descriptors_without_a_device_report_hip_error(lib):
    import torch

    if torch.cuda.is_available():
        pytest.skip("a device is present")
    st, h = _create(lib, [_desc(), _desc(dim=128, dtype=eb.EB_INT8_ROWWISE),
                          _desc(dim=128, dtype=eb.EB_INT8_ROWWISE_SPLIT)])
    assert st == eb.EB_ERR_HIP and h is None


def test_binding_fails_loudly_without_the_library(tmp_path):
    with pytest.raises(RuntimeError, match="not found"):
        saved = eb._lib
        eb._lib = None
        try:
            eb.load_library(str(tmp_path / "missing.so"))
        finally:
            eb._lib = saved


def test_binding_refuses_host_tensors(lib):
    # the kernels read these pointers directly: a host tensor must never reach them
    import torch

    with pytest.raises(ValueError, match="device tensors"):
        eb.eb_create_tables([(torch.zeros(10, 16), 16, "f32")])
    h = eb.EbTables(None, [], None, 16, torch.device("cuda:0"))
    idx, off = torch.zeros(4, dtype=torch.int64), torch.tensor([0, 2, 4])
    out = torch.empty(2, 16)
    with pytest.raises(ValueError, match="handle's GPU"):
        eb.eb_forward(h, idx, off, None, "sum", out)
    with pytest.raises(ValueError, match="handle's GPU"):
        eb.eb_forward_seq(h, idx, off, torch.empty(64))
    with pytest.raises(ValueError, match="handle's GPU"):
        eb.eb_fm_cross(h, out, torch.empty(2))
    with pytest.raises(ValueError, match="handle's GPU"):
        eb.eb_backward_update(h, idx, off, None, "sum", out, workspace=torch.empty(8, dtype=torch.uint8))
