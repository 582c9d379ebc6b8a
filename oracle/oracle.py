"""ctypes marshalling for the plain-C oracle (test infrastructure only).

The oracle computes, for every requested bag g = t*B + b, the fp64 sum
S[d] = sum_i w_i * x(t, idx_i, d) rounded once to fp32 (divided by the bag
length first for mean pooling; +0.0 for an empty bag) — the definition of the
pooled embedding lookup of the paper's sparse_arch (Sec. IV-A.2) over jagged
categorical features (Abstract, Sec. IV-A.3).  See eb_oracle.c.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "eb_oracle.c")
_LIB_NAME = "libeb_oracle.so"

_ROW_CODES = {"f32": 0, "f16": 1, "int8_rowwise": 2, "int8_rowwise_split": 3}
_MODE_CODES = {"sum": 0, "mean": 1}
_ERRORS = {-1: "invalid argument", -2: "dtype", -3: "shape", -5: "index out of range", -6: "bad offsets"}


class OracleError(RuntimeError):
    def __init__(self, code: int):
        super().__init__(f"oracle error {code}: {_ERRORS.get(code, 'unknown')}")
        self.code = code


# EBO_ORACLE_LIB names another build of eb_oracle.c to load (the sanitizer
# build of the tests); by default the library built next to the source.
_LIB_ENV = "EBO_ORACLE_LIB"

# AddressSanitizer and UndefinedBehaviorSanitizer, every report fatal.
SANITIZE_FLAGS = ["-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                  "-fno-omit-frame-pointer"]


def lib_path() -> str:
    return os.environ.get(_LIB_ENV) or os.path.join(_HERE, _LIB_NAME)


def build(out: Optional[str] = None, sanitize: bool = False) -> str:
    """Compile eb_oracle.c with gcc (-O2, no fast-math, no FP contraction,
    OpenMP) into `out` (default: lib_path()).  sanitize=True builds it with
    AddressSanitizer and UndefinedBehaviorSanitizer instead of -O2; such a
    library must be loaded into a process that preloads the ASan runtime."""
    out = out or lib_path()
    tmp = out + ".tmp"
    opt = SANITIZE_FLAGS if sanitize else ["-O2"]
    cmd = ["gcc", *opt, "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
           "-Wall", "-Wextra", "-shared", "-fPIC", "-o", tmp, _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


class _CTable(ctypes.Structure):
    _fields_ = [
        ("data", ctypes.c_void_p),
        ("num_rows", ctypes.c_int64),
        ("dim", ctypes.c_int32),
        ("dtype", ctypes.c_int32),
        ("row_stride_bytes", ctypes.c_int64),
    ]


_lib = None


def _load():
    global _lib
    if _lib is None:
        path = lib_path()
        if not os.environ.get(_LIB_ENV) and (not os.path.exists(path) or
                                             os.path.getmtime(path) < os.path.getmtime(_SRC)):
            build()
        lib = ctypes.CDLL(path)
        lib.ebo_forward.restype = ctypes.c_int
        lib.ebo_forward.argtypes = [
            ctypes.POINTER(_CTable), ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
            ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p,
            ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int32,
        ]
        lib.ebo_half_to_double.restype = ctypes.c_double
        lib.ebo_half_to_double.argtypes = [ctypes.c_uint16]
        lib.ebo_max_threads.restype = ctypes.c_int
        lib.ebo_max_threads.argtypes = []
        lib.ebo_double_to_half.restype = ctypes.c_uint16
        lib.ebo_double_to_half.argtypes = [ctypes.c_double]
        lib.ebo_backward_update.restype = ctypes.c_int
        lib.ebo_backward_update.argtypes = [
            ctypes.POINTER(_CTable), ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
            ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p, ctypes.c_int32,
            ctypes.c_float, ctypes.c_float, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
        ]
        lib.ebo_forward_seq.restype = ctypes.c_int
        lib.ebo_forward_seq.argtypes = [
            ctypes.POINTER(_CTable), ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
            ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32,
        ]
        lib.ebo_fm.restype = ctypes.c_int
        lib.ebo_fm.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int64,
                               ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32]
        _lib = lib
    return _lib


@dataclass
class OracleTable:
    """Host rows of one table: `rows` is a C-contiguous numpy array whose first
    axis is the row (its byte stride is the row stride), or None when no bag
    that is asked for reads this table (then num_rows must be given).

    For "int8_rowwise_split" the table is one byte buffer: num_rows rows of
    codes at row_stride bytes apart, then the rows' 4-byte scale/bias words;
    `rows` is that whole buffer (any shape, C-contiguous) and num_rows and
    row_stride must be given."""

    rows: Optional[np.ndarray]
    dim: int
    dtype: str
    num_rows: Optional[int] = None
    row_stride: Optional[int] = None

    @classmethod
    def of(cls, table, with_rows: bool = True) -> "OracleTable":
        """The oracle's view of a table object with host_bytes(), dim, dtype,
        num_rows and row_stride_bytes (the seeded input generator's Table):
        a host copy of its bytes, or only its shape when with_rows is False."""
        rows = table.host_bytes() if with_rows else None
        stride = table.row_stride_bytes if table.dtype == "int8_rowwise_split" else None
        return cls(rows, table.dim, table.dtype, table.num_rows, stride)


def _fill_table(ct, tb: OracleTable, need_rows: bool = False, writable: bool = False):
    """Marshal one OracleTable into the oracle's C struct."""
    if tb.rows is None:
        if need_rows:
            raise ValueError("this oracle call reads every table's rows")
        ct.data = None
        ct.num_rows = int(tb.num_rows)
        ct.row_stride_bytes = 0
    else:
        if not tb.rows.flags["C_CONTIGUOUS"] or (writable and not tb.rows.flags["WRITEABLE"]):
            raise ValueError("table rows must be C-contiguous" + (" and writable" if writable else ""))
        ct.data = tb.rows.ctypes.data
        if tb.dtype == "int8_rowwise_split":
            if tb.num_rows is None or tb.row_stride is None:
                raise ValueError("a split int8 table needs num_rows and row_stride")
            if tb.rows.nbytes < int(tb.num_rows) * (int(tb.row_stride) + 4):
                raise ValueError("a split int8 table's buffer must hold the codes and the scale/bias block")
            ct.num_rows = int(tb.num_rows)
            ct.row_stride_bytes = int(tb.row_stride)
        else:
            ct.num_rows = tb.rows.shape[0]
            ct.row_stride_bytes = tb.rows.strides[0]
    ct.dim = int(tb.dim)
    ct.dtype = _ROW_CODES[tb.dtype]


def half_to_double(bits: int) -> float:
    """The oracle's binary16 decoder (exposed so tests can pin it)."""
    return float(_load().ebo_half_to_double(int(bits) & 0xFFFF))


def max_threads() -> int:
    return int(_load().ebo_max_threads())


def ebo_forward(
    tables: Sequence[OracleTable],
    indices: np.ndarray,
    offsets: np.ndarray,
    weights: Optional[np.ndarray] = None,
    pooling: str = "sum",
    bags: Optional[np.ndarray] = None,
    num_threads: int = 0,
    with_absum: bool = False,
):
    """Run the oracle.  Returns out (fp32) or (out, absum) with absum fp64.

    bags is None: out is [B, sum D].  Otherwise out is [len(bags), max D] and
    row k holds bag bags[k] in its first D_t columns.
    """
    lib = _load()
    offsets = np.ascontiguousarray(offsets)
    indices = np.ascontiguousarray(indices)
    if offsets.dtype == np.int64:
        itype = 1
    elif offsets.dtype == np.int32:
        itype = 0
    else:
        raise TypeError("offsets must be int32 or int64")
    if indices.dtype != offsets.dtype:
        raise TypeError("indices and offsets must share a dtype")
    ct = (_CTable * len(tables))()
    for i, tb in enumerate(tables):
        _fill_table(ct[i], tb)
    T = len(tables)
    nbags = offsets.size - 1
    B = nbags // T if T else 0
    sum_d = sum(int(t.dim) for t in tables)
    if weights is not None:
        weights = np.ascontiguousarray(weights, dtype=np.float32)
    if bags is None:
        out = np.empty((B, sum_d), dtype=np.float32)
        ld = sum_d
        bag_ptr, nsel = None, 0
    else:
        bags = np.ascontiguousarray(bags, dtype=np.int64)
        ld = max(int(t.dim) for t in tables)
        out = np.empty((bags.size, ld), dtype=np.float32)
        bag_ptr, nsel = bags.ctypes.data, bags.size
    absum = np.empty(out.shape, dtype=np.float64) if with_absum else None
    rc = lib.ebo_forward(
        ct, T, indices.ctypes.data if indices.size else None, offsets.ctypes.data, itype, indices.size,
        offsets.size, weights.ctypes.data if weights is not None else None, _MODE_CODES[pooling],
        bag_ptr, nsel, out.ctypes.data, ld if bags is not None else 0,
        absum.ctypes.data if absum is not None else None, int(num_threads),
    )
    if rc != 0:
        raise OracleError(rc)
    return (out, absum) if with_absum else out


class _CReport(ctypes.Structure):
    _fields_ = [
        ("rows", ctypes.c_void_p),
        ("grad", ctypes.c_void_p),
        ("scale", ctypes.c_void_p),
        ("count", ctypes.c_void_p),
        ("num_rows", ctypes.c_int64),
    ]


_OPT_CODES = {"sgd": 0, "rowwise_adagrad": 1}


def double_to_half(x: float) -> int:
    """The oracle's fp64 -> binary16 rounding (exposed so tests can pin it)."""
    return int(_load().ebo_double_to_half(float(x)))


def ebo_backward_update(
    tables: Sequence[OracleTable],
    indices: np.ndarray,
    offsets: np.ndarray,
    weights: Optional[np.ndarray],
    pooling: str,
    grad_out: np.ndarray,
    optimizer: str = "sgd",
    lr: float = 0.01,
    eps: float = 1e-8,
    state: Optional[np.ndarray] = None,
    report=(),
    num_threads: int = 0,
):
    """Backward of the pooled lookup plus the fused optimizer step, in place.

    Updates each table's rows (tables whose rows are None are skipped) and,
    for row-wise Adagrad, `state` (fp32 [sum_t R_t]).  `report` lists tables
    whose touched rows to return as {t: (rows, grad, scale, count)}.
    """
    lib = _load()
    offsets = np.ascontiguousarray(offsets)
    indices = np.ascontiguousarray(indices)
    itype = 1 if offsets.dtype == np.int64 else 0
    if indices.dtype != offsets.dtype:
        raise TypeError("indices and offsets must share a dtype")
    grad_out = np.ascontiguousarray(grad_out, dtype=np.float32)
    T = len(tables)
    ct = (_CTable * T)()
    for i, tb in enumerate(tables):
        _fill_table(ct[i], tb, writable=True)
    B = (offsets.size - 1) // T
    lens = [int(offsets[(t + 1) * B] - offsets[t * B]) for t in range(T)]
    reps = (_CReport * T)()
    keep = {}
    for t in report:
        n = max(lens[t], 1)
        D = int(tables[t].dim)
        arrs = (np.zeros(n, np.int64), np.zeros((n, D), np.float64), np.zeros((n, D), np.float64),
                np.zeros(n, np.int64))
        keep[t] = arrs
        reps[t].rows, reps[t].grad, reps[t].scale, reps[t].count = [a.ctypes.data for a in arrs]
    if weights is not None:
        weights = np.ascontiguousarray(weights, dtype=np.float32)
    if state is not None:
        assert state.dtype == np.float32 and state.flags["C_CONTIGUOUS"]
    rc = lib.ebo_backward_update(
        ct, T, indices.ctypes.data if indices.size else None, offsets.ctypes.data, itype, indices.size,
        offsets.size, weights.ctypes.data if weights is not None else None, _MODE_CODES[pooling],
        grad_out.ctypes.data, _OPT_CODES[optimizer], float(lr), float(eps),
        state.ctypes.data if state is not None else None, reps, int(num_threads),
    )
    if rc != 0:
        raise OracleError(rc)
    out = {}
    for t, (rows, g, s, c) in keep.items():
        n = int(reps[t].num_rows)
        out[t] = (rows[:n], g[:n], s[:n], c[:n])
    return out


def ebo_fm(pooled: np.ndarray, num_fields: int, dim: int, asum: Optional[np.ndarray] = None,
           num_threads: int = 0):
    """Factorization-machine cross term of each example over its pooled field
    embeddings: y[b] = sum_{f<f'} <e_{b,f}, e_{b,f'}> in fp64 (see eb_oracle.c).

    pooled: fp32 [B, ld >= num_fields * dim], field f in columns [f*dim, (f+1)*dim).
    Returns y (fp64 [B]), or (y, scale) when asum (fp64, pooled's shape) is given.
    """
    lib = _load()
    pooled = np.ascontiguousarray(pooled, dtype=np.float32)
    if pooled.ndim != 2:
        raise ValueError("pooled must be 2-D")
    B, ld = pooled.shape
    y = np.empty(B, np.float64)
    scale = None
    if asum is not None:
        asum = np.ascontiguousarray(asum, dtype=np.float64)
        if asum.shape != pooled.shape:
            raise ValueError("asum must have pooled's shape")
        scale = np.empty(B, np.float64)
    rc = lib.ebo_fm(pooled.ctypes.data, ld, int(num_fields), int(dim), B,
                    asum.ctypes.data if asum is not None else None, y.ctypes.data,
                    scale.ctypes.data if scale is not None else None, int(num_threads))
    if rc != 0:
        raise OracleError(rc)
    return y if scale is None else (y, scale)


def ebo_forward_seq(tables: Sequence[OracleTable], indices: np.ndarray, offsets: np.ndarray,
                    out_numel: Optional[int] = None, num_threads: int = 0) -> np.ndarray:
    """Un-pooled lookup: every position's row as fp32, table t's positions as a
    [N_t, D_t] block, blocks in table order (see eb_oracle.c).  Returns the flat
    fp32 array; out_numel defaults to sum_t N_t * D_t."""
    lib = _load()
    offsets = np.ascontiguousarray(offsets)
    indices = np.ascontiguousarray(indices)
    if offsets.dtype not in (np.int32, np.int64) or indices.dtype != offsets.dtype:
        raise TypeError("indices and offsets must share an int32 or int64 dtype")
    T = len(tables)
    ct = (_CTable * T)()
    for i, tb in enumerate(tables):
        _fill_table(ct[i], tb, need_rows=True)
    if out_numel is None:
        B = (offsets.size - 1) // T
        out_numel = sum(int(offsets[(t + 1) * B] - offsets[t * B]) * int(tables[t].dim) for t in range(T))
    out = np.empty(max(int(out_numel), 0), np.float32)
    rc = lib.ebo_forward_seq(ct, T, indices.ctypes.data if indices.size else None, offsets.ctypes.data,
                             1 if offsets.dtype == np.int64 else 0, indices.size, offsets.size,
                             out.ctypes.data if out.size else None, int(out_numel), int(num_threads))
    if rc != 0:
        raise OracleError(rc)
    return out
