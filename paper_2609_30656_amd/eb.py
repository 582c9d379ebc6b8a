"""Python binding of libeb — argument marshalling only.

Each function has the name of the C entry point it calls (include/eb.h) and
turns torch tensors into the plain pointers and sizes the C ABI takes.  Every
step of the lookups, the FM term and the backward runs in libeb's HIP
kernels; torch only owns the device memory and the stream.  If libeb.so has not been built this module
raises on first use: there is no other implementation to fall back to.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libeb.so")

# eb_status
EB_OK = 0
EB_ERR_INVALID_ARG = -1
EB_ERR_DTYPE = -2
EB_ERR_SHAPE = -3
EB_ERR_UNSUPPORTED = -4
EB_ERR_INDEX_OOB = -5
EB_ERR_OFFSETS = -6
EB_ERR_OOM = -7
EB_ERR_HIP = -8
# eb_table_dtype
EB_F32, EB_F16, EB_INT8_ROWWISE, EB_INT8_ROWWISE_SPLIT = 0, 1, 2, 3
# eb_elem_type
EB_I32, EB_I64, EB_T_F32 = 0, 1, 2
# eb_pooling
EB_POOL_SUM, EB_POOL_MEAN = 0, 1
# eb_optimizer
EB_OPT_SGD, EB_OPT_ROWWISE_ADAGRAD = 0, 1

TABLE_DTYPES = {"f32": EB_F32, "f16": EB_F16, "int8_rowwise": EB_INT8_ROWWISE,
                "int8_rowwise_split": EB_INT8_ROWWISE_SPLIT}
POOLING = {"sum": EB_POOL_SUM, "mean": EB_POOL_MEAN}
OPTIMIZERS = {"sgd": EB_OPT_SGD, "rowwise_adagrad": EB_OPT_ROWWISE_ADAGRAD}
EXPORTED = ("eb_create_tables", "eb_forward", "eb_forward_seq", "eb_fm_cross", "eb_forward_fm", "eb_destroy",
            "eb_status_string", "eb_backward_workspace_size", "eb_backward_update", "eb_backward_update_noalloc")
# bytes of the static workspace of eb_backward_update_noalloc
EB_NOALLOC_SCRATCH_BYTES = 128 << 20


class EBError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: {eb_status_string(status)} ({status})")
        self.status = status


class eb_table_desc(ctypes.Structure):
    _fields_ = [
        ("data", ctypes.c_void_p),
        ("num_rows", ctypes.c_int64),
        ("dim", ctypes.c_int32),
        ("dtype", ctypes.c_int32),
        ("row_stride_bytes", ctypes.c_int64),
    ]


class eb_tensor(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("numel", ctypes.c_int64), ("elem_type", ctypes.c_int32)]


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libeb.so (once).  Raises if it is missing: build it first."""
    global _lib
    if _lib is None:
        if not os.path.exists(path):
            raise RuntimeError(f"libeb.so not found at {path}; build it with "
                               "`python -c 'import __graft_entry__ as g; g.build()'`")
        lib = ctypes.CDLL(path)
        lib.eb_create_tables.restype = ctypes.c_int
        lib.eb_create_tables.argtypes = [ctypes.POINTER(eb_table_desc), ctypes.c_int32, ctypes.c_void_p,
                                         ctypes.POINTER(ctypes.c_void_p)]
        lib.eb_forward.restype = ctypes.c_int
        lib.eb_forward.argtypes = [ctypes.c_void_p, eb_tensor, eb_tensor, eb_tensor, ctypes.c_int, eb_tensor]
        lib.eb_forward_fm.restype = ctypes.c_int
        lib.eb_forward_fm.argtypes = [ctypes.c_void_p, eb_tensor, eb_tensor, eb_tensor, ctypes.c_int, eb_tensor,
                                      eb_tensor]
        lib.eb_forward_seq.restype = ctypes.c_int
        lib.eb_forward_seq.argtypes = [ctypes.c_void_p, eb_tensor, eb_tensor, eb_tensor]
        lib.eb_fm_cross.restype = ctypes.c_int
        lib.eb_fm_cross.argtypes = [ctypes.c_void_p, eb_tensor, eb_tensor]
        lib.eb_destroy.restype = ctypes.c_int
        lib.eb_destroy.argtypes = [ctypes.c_void_p]
        lib.eb_status_string.restype = ctypes.c_char_p
        lib.eb_status_string.argtypes = [ctypes.c_int]
        lib.eb_backward_workspace_size.restype = ctypes.c_int
        lib.eb_backward_workspace_size.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.POINTER(ctypes.c_size_t)]
        lib.eb_backward_update.restype = ctypes.c_int
        lib.eb_backward_update.argtypes = [ctypes.c_void_p, eb_tensor, eb_tensor, eb_tensor, ctypes.c_int, eb_tensor,
                                           ctypes.c_int32, ctypes.c_float, ctypes.c_float, eb_tensor,
                                           ctypes.c_void_p, ctypes.c_size_t]
        lib.eb_backward_update_noalloc.restype = ctypes.c_int
        lib.eb_backward_update_noalloc.argtypes = [ctypes.c_void_p, eb_tensor, eb_tensor, eb_tensor, ctypes.c_int,
                                                   eb_tensor, ctypes.c_int32, ctypes.c_float, ctypes.c_float,
                                                   eb_tensor]
        _lib = lib
    return _lib


def eb_status_string(status: int) -> str:
    return load_library().eb_status_string(int(status)).decode()


class EbTables:
    """Handle returned by eb_create_tables; keeps the table tensors alive."""

    def __init__(self, ptr: int, tables, stream, sum_dim: int, device: Optional[torch.device] = None):
        self.ptr = ptr
        self.tables = list(tables)
        self.stream = stream
        self.sum_dim = sum_dim
        self.device = device

    @property
    def num_tables(self) -> int:
        return len(self.tables)

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        eb_destroy(self)


def _torch_stream(stream, device: torch.device) -> torch.cuda.Stream:
    """The handle's stream as a torch stream (None: the null stream)."""
    if stream is None or (isinstance(stream, int) and stream == 0):
        return torch.cuda.default_stream(device)
    if isinstance(stream, int):
        return torch.cuda.ExternalStream(stream, device=device)
    return stream


def _stream_handle(stream) -> Optional[int]:
    if stream is None:
        return None
    if isinstance(stream, int):
        return stream or None
    return stream.cuda_stream or None


def eb_create_tables(tables: Sequence, stream=None) -> EbTables:
    """tables: objects with .rows (device tensor, first axis = row), .dim and
    .dtype ("f32" | "f16" | "int8_rowwise" | "int8_rowwise_split"), or
    (rows, dim, dtype) tuples.  A split int8 table's rows view the codes of
    an allocation whose scale/bias block follows them.
    stream: torch.cuda.Stream, raw hipStream_t as int, or None (null stream)."""
    lib = load_library()
    norm = []
    for t in tables:
        rows, dim, dtype = (t.rows, t.dim, t.dtype) if hasattr(t, "rows") else t
        norm.append((rows, int(dim), dtype))
    devices = {r.device for r, _, _ in norm}
    if any(d.type != "cuda" for d in devices) or len(devices) > 1:
        raise ValueError(f"eb tables must be device tensors of one GPU, got {sorted(map(str, devices))}")
    descs = (eb_table_desc * len(norm))()
    for i, (rows, dim, dtype) in enumerate(norm):
        descs[i].data = rows.data_ptr() if rows.numel() else None
        descs[i].num_rows = rows.shape[0]
        descs[i].dim = dim
        descs[i].dtype = TABLE_DTYPES[dtype] if isinstance(dtype, str) else int(dtype)
        descs[i].row_stride_bytes = rows.stride(0) * rows.element_size()
        if descs[i].dtype == EB_INT8_ROWWISE_SPLIT:
            # the kernels read the scale/bias block after the rows' codes:
            # it must lie inside the memory that `rows` views
            need = rows.shape[0] * (descs[i].row_stride_bytes + 4)
            have = rows.untyped_storage().nbytes() - rows.storage_offset() * rows.element_size()
            if have < need:
                raise ValueError(f"a split int8 table needs {need} bytes from its first row (codes, then the "
                                 f"scale/bias block), its storage holds {have}")
    out = ctypes.c_void_p()
    st = lib.eb_create_tables(descs, len(norm), _stream_handle(stream), ctypes.byref(out))
    if st != EB_OK:
        raise EBError(st, "eb_create_tables")
    return EbTables(out.value, [r for r, _, _ in norm], stream, sum(d for _, d, _ in norm),
                    norm[0][0].device if norm else None)


_ELEM = {torch.int32: EB_I32, torch.int64: EB_I64, torch.float32: EB_T_F32}


def _as_tensor(t: Optional[torch.Tensor], device: Optional[torch.device] = None) -> eb_tensor:
    """The eb_tensor view of a contiguous device tensor (of `device`, the
    handle's GPU, when given): the kernels read these pointers directly, so a
    host tensor is refused here rather than handed to the GPU."""
    if t is None:
        return eb_tensor(None, 0, EB_T_F32)
    if not t.is_contiguous():
        raise ValueError("eb tensors must be contiguous")
    if t.device.type != "cuda" or (device is not None and t.device != device):
        raise ValueError(f"eb tensors must be on the handle's GPU ({device}), got one on {t.device}")
    return eb_tensor(t.data_ptr() if t.numel() else None, t.numel(), _ELEM.get(t.dtype, 99))


def eb_forward(tables: EbTables, indices: torch.Tensor, offsets: torch.Tensor,
               per_sample_weights: Optional[torch.Tensor], pooling, out: torch.Tensor) -> torch.Tensor:
    """Enqueue the pooled lookup on the handle's stream; returns `out`."""
    lib = load_library()
    mode = POOLING[pooling] if isinstance(pooling, str) else int(pooling)
    d = tables.device
    st = lib.eb_forward(tables.ptr, _as_tensor(indices, d), _as_tensor(offsets, d),
                        _as_tensor(per_sample_weights, d), mode, _as_tensor(out, d))
    if st != EB_OK:
        raise EBError(st, "eb_forward")
    return out


def eb_forward_seq(tables: EbTables, indices: torch.Tensor, offsets: torch.Tensor, out: torch.Tensor) -> torch.Tensor:
    """Un-pooled lookup: every position's row as fp32 into out (table t's
    positions as a [N_t, D_t] block, blocks in table order); returns out."""
    d = tables.device
    st = load_library().eb_forward_seq(tables.ptr, _as_tensor(indices, d), _as_tensor(offsets, d), _as_tensor(out, d))
    if st != EB_OK:
        raise EBError(st, "eb_forward_seq")
    return out


def eb_fm_cross(tables: EbTables, pooled: torch.Tensor, fm_out: torch.Tensor) -> torch.Tensor:
    """FM cross term of each example of a pooled output [B, T*D] into fm_out [B]; returns fm_out."""
    d = tables.device
    st = load_library().eb_fm_cross(tables.ptr, _as_tensor(pooled, d), _as_tensor(fm_out, d))
    if st != EB_OK:
        raise EBError(st, "eb_fm_cross")
    return fm_out


def eb_forward_fm(tables: EbTables, indices: torch.Tensor, offsets: torch.Tensor,
                  per_sample_weights: Optional[torch.Tensor], pooling, out: torch.Tensor,
                  fm_out: torch.Tensor) -> torch.Tensor:
    """eb_forward, then eb_fm_cross on its output into fm_out [B]; returns fm_out."""
    lib = load_library()
    mode = POOLING[pooling] if isinstance(pooling, str) else int(pooling)
    d = tables.device
    st = lib.eb_forward_fm(tables.ptr, _as_tensor(indices, d), _as_tensor(offsets, d),
                           _as_tensor(per_sample_weights, d), mode, _as_tensor(out, d), _as_tensor(fm_out, d))
    if st != EB_OK:
        raise EBError(st, "eb_forward_fm")
    return fm_out


def eb_destroy(tables: EbTables) -> None:
    if tables.ptr:
        st = load_library().eb_destroy(tables.ptr)
        tables.ptr = None
        if st != EB_OK:
            raise EBError(st, "eb_destroy")


def eb_backward_workspace_size(tables: EbTables, num_indices: int) -> int:
    n = ctypes.c_size_t()
    st = load_library().eb_backward_workspace_size(tables.ptr, int(num_indices), ctypes.byref(n))
    if st != EB_OK:
        raise EBError(st, "eb_backward_workspace_size")
    return int(n.value)


def eb_backward_update(tables: EbTables, indices: torch.Tensor, offsets: torch.Tensor,
                       per_sample_weights: Optional[torch.Tensor], pooling, grad_out: torch.Tensor,
                       optimizer="sgd", learning_rate: float = 0.01, eps: float = 1e-8,
                       optimizer_state: Optional[torch.Tensor] = None,
                       workspace: Optional[torch.Tensor] = None) -> None:
    """Enqueue the backward + optimizer step on the handle's stream.

    workspace: a contiguous device tensor (any element type) of at least
    eb_backward_workspace_size() bytes that stays untouched until the step
    has run on the handle's stream; when None, one is allocated on that
    stream (torch's allocator then reuses it only for work ordered after the
    step on the same stream)."""
    lib = load_library()
    d = tables.device
    args = (_as_tensor(indices, d), _as_tensor(offsets, d), _as_tensor(per_sample_weights, d))
    g, st_t = _as_tensor(grad_out, d), _as_tensor(optimizer_state, d)
    if workspace is None:
        nbytes = eb_backward_workspace_size(tables, indices.numel())
        with torch.cuda.stream(_torch_stream(tables.stream, d)):
            workspace = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=d)
    elif workspace.device != d:
        raise ValueError(f"the workspace must be on the handle's GPU ({d}), got one on {workspace.device}")
    elif not workspace.is_contiguous():
        raise ValueError("the workspace must be contiguous")
    mode = POOLING[pooling] if isinstance(pooling, str) else int(pooling)
    opt = OPTIMIZERS[optimizer] if isinstance(optimizer, str) else int(optimizer)
    st = lib.eb_backward_update(tables.ptr, *args, mode, g, opt, float(learning_rate), float(eps),
                                st_t, workspace.data_ptr(), workspace.numel() * workspace.element_size())
    if st != EB_OK:
        raise EBError(st, "eb_backward_update")


def eb_backward_update_noalloc(tables: EbTables, indices: torch.Tensor, offsets: torch.Tensor,
                               per_sample_weights: Optional[torch.Tensor], pooling, grad_out: torch.Tensor,
                               optimizer="sgd", learning_rate: float = 0.01, eps: float = 1e-8,
                               optimizer_state: Optional[torch.Tensor] = None) -> None:
    """eb_backward_update with the library's static workspace: allocates
    nothing (EB_ERR_UNSUPPORTED if the batch needs more than
    EB_NOALLOC_SCRATCH_BYTES of workspace).  Calls that overlap on one GPU
    race on that workspace."""
    lib = load_library()
    d = tables.device
    args = (_as_tensor(indices, d), _as_tensor(offsets, d), _as_tensor(per_sample_weights, d))
    g, st_t = _as_tensor(grad_out, d), _as_tensor(optimizer_state, d)
    mode = POOLING[pooling] if isinstance(pooling, str) else int(pooling)
    opt = OPTIMIZERS[optimizer] if isinstance(optimizer, str) else int(optimizer)
    st = lib.eb_backward_update_noalloc(tables.ptr, *args, mode, g, opt, float(learning_rate), float(eps), st_t)
    if st != EB_OK:
        raise EBError(st, "eb_backward_update_noalloc")
