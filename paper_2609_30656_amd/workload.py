"""Seeded synthetic inputs shaped like the paper's recommendation workloads.

The paper profiles a DLRM whose sparse_arch looks up embedding tables over
jagged categorical features (Sec. IV-A.2) and stresses that the sparsity of
those features drives performance (Sec. I) and that inputs should keep the
real distribution (Sec. III-B.1, batch replication).  Its data is not
available, so every input here is drawn from seeded distributions with the
shapes of the five workloads this library is measured on (table count, rows,
dim, storage type, batch, bag-length law, index law, pooling mode).

This module draws tables, lengths, indices and weights only; it holds none of
the pooling arithmetic, and both the GPU path and the CPU oracle consume what
it produces.  Scalar choices (dims, row counts, which tables are one-hot, the
Zipf rank->row permutation) come from numpy's seeded generator and are the
same on every machine; bulk arrays come from a seeded torch generator on the
device they live on (CPU or GPU), so they are reproducible per device.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Callable, List, Optional

import numpy as np
import torch

SEED_ROOT = 2609

# storage formats (names shared by the binding and the oracle wrapper)
F32 = "f32"
F16 = "f16"
INT8_ROWWISE = "int8_rowwise"
INT8_ROWWISE_SPLIT = "int8_rowwise_split"
INT8_DTYPES = (INT8_ROWWISE, INT8_ROWWISE_SPLIT)
# int8 row layouts: "packed" = codes then the fp16 scale and bias in each row
# (D + 4 bytes); "split" = codes only in the rows, the rows' scale/bias words
# in one block after them
INT8_LAYOUTS = {"packed": INT8_ROWWISE, "split": INT8_ROWWISE_SPLIT}


@dataclass
class Table:
    """One embedding table: `rows` is a [R, ...] tensor whose first axis is the row.

    For f32/f16 it is [R, D] of that dtype; for int8_rowwise it is [R, stride]
    uint8 holding D codes, an fp16 scale and an fp16 bias per row.  For
    int8_rowwise_split, `storage` is the table's whole byte buffer (R rows of
    `stride` bytes holding the D codes, then R 4-byte scale/bias words) and
    `rows` the [R, stride] view of its codes.
    """

    rows: torch.Tensor
    dim: int
    dtype: str
    storage: Optional[torch.Tensor] = None

    @property
    def num_rows(self) -> int:
        return int(self.rows.shape[0])

    @property
    def row_stride_bytes(self) -> int:
        return int(self.rows.stride(0) * self.rows.element_size())

    @property
    def row_bytes(self) -> int:
        """Bytes of one row that a lookup reads (codes + scale/bias for int8)."""
        return 4 * self.dim if self.dtype == F32 else (2 * self.dim if self.dtype == F16 else self.dim + 4)

    def host_bytes(self):
        """A host (numpy) copy of the table's memory: the rows, or for the
        split int8 layout the whole buffer (codes, then scale/bias block)."""
        src = self.storage if self.dtype == INT8_ROWWISE_SPLIT else self.rows
        return src.detach().cpu().numpy()

    def clone(self) -> "Table":
        """A copy of the table in new memory on the same device."""
        if self.dtype == INT8_ROWWISE_SPLIT:
            st = self.storage.clone()
            R, stride = self.num_rows, self.row_stride_bytes
            return Table(st[:R * stride].view(R, stride), self.dim, self.dtype, st)
        return Table(self.rows.clone(), self.dim, self.dtype)


@dataclass
class Workload:
    name: str
    tables: List[Table]
    batch: int
    indices: torch.Tensor  # int64 or int32 [N], table-major
    offsets: torch.Tensor  # same dtype, [T*B + 1]
    weights: Optional[torch.Tensor]  # fp32 [N] or None
    pooling: str  # "sum" | "mean"
    lengths: torch.Tensor = field(repr=False, default=None)  # int64 [T*B]

    @property
    def num_tables(self) -> int:
        return len(self.tables)

    @property
    def num_bags(self) -> int:
        return self.num_tables * self.batch

    @property
    def num_indices(self) -> int:
        return int(self.indices.numel())

    @property
    def sum_dim(self) -> int:
        return sum(t.dim for t in self.tables)

    def algorithmic_bytes(self) -> int:
        """Bytes one forward must move at minimum by the metric's definition.

        Gathered row bytes (every lookup, duplicates counted) + index bytes +
        offset bytes + weight bytes + output bytes.
        """
        esz = self.indices.element_size()
        lens = self.lengths.view(self.num_tables, self.batch).sum(dim=1).cpu().tolist()
        row = sum(int(n) * t.row_bytes for n, t in zip(lens, self.tables))
        idx = self.num_indices * esz
        off = int(self.offsets.numel()) * esz
        w = self.num_indices * 4 if self.weights is not None else 0
        out = self.batch * self.sum_dim * 4
        return row + idx + off + w + out

    def table_lookups(self) -> List[int]:
        """Number of index positions of each table."""
        return [int(n) for n in self.lengths.view(self.num_tables, self.batch).sum(dim=1).cpu().tolist()]

    def seq_output_numel(self) -> int:
        """fp32 elements of the un-pooled lookup's output (a D_t row per position)."""
        return sum(n * t.dim for n, t in zip(self.table_lookups(), self.tables))

    def seq_algorithmic_bytes(self) -> int:
        """Bytes one un-pooled lookup must move at minimum: each position's row
        read, its index read and its fp32 row written, plus the T + 1 table
        starts of the offsets."""
        esz = self.indices.element_size()
        total = (self.num_tables + 1) * esz
        for n, t in zip(self.table_lookups(), self.tables):
            total += n * (t.row_bytes + esz + 4 * t.dim)
        return total

    def backward_algorithmic_bytes(self) -> int:
        """Bytes one backward + row-wise Adagrad step must move at minimum: the
        gathered gradient rows (4*D per lookup), each touched table row read and
        written once, its optimizer state read and written once, and the
        indices, offsets and weights."""
        esz = self.indices.element_size()
        total = self.num_indices * esz + int(self.offsets.numel()) * esz
        if self.weights is not None:
            total += self.num_indices * 4
        off = self.offsets.cpu()
        B = self.batch
        for t, tb in enumerate(self.tables):
            lo, hi = int(off[t * B]), int(off[(t + 1) * B])
            u = int(torch.unique(self.indices[lo:hi]).numel()) if hi > lo else 0
            total += (hi - lo) * 4 * tb.dim + u * (2 * tb.row_bytes + 8)
        return total


def _seed(*parts: int) -> int:
    """63-bit torch seed derived from a tuple of small integers."""
    ss = np.random.SeedSequence([SEED_ROOT, *[int(p) for p in parts]])
    return int(ss.generate_state(1, np.uint64)[0] & np.uint64((1 << 63) - 1))


def _np_rng(*parts: int) -> np.random.Generator:
    return np.random.default_rng([SEED_ROOT, *[int(p) for p in parts]])


def _torch_gen(device: torch.device, *parts: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(_seed(*parts))
    return g


# stream ids of the seed tuple (config, table, stream, batch_seed)
_S_VALUES, _S_LENGTHS, _S_INDICES, _S_WEIGHTS, _S_PARAMS = 0, 1, 2, 3, 4

# ----------------------------------------------------------------------------
# value distributions


def _values_uniform_f32(R, D, gen, device):
    return torch.rand((R, D), generator=gen, device=device, dtype=torch.float32).mul_(2.0).sub_(1.0)


def _values_normal(R, D, gen, device, dtype):
    # N(0, 0.01), rounded once to the storage type (fp16 keeps subnormals and -0.0)
    v = torch.randn((R, D), generator=gen, device=device, dtype=torch.float32).mul_(0.01)
    return v.to(dtype)


def _values_int8_rowwise(R, D, gen, device, stride):
    """Uniform codes 0..255, scale ~ U(1e-4, 4e-4), bias ~ U(-0.06, -0.02), both fp16."""
    rows = torch.empty((R, stride), dtype=torch.uint8, device=device)
    rows[:, :D] = torch.randint(0, 256, (R, D), generator=gen, device=device, dtype=torch.uint8)
    scale = torch.rand((R,), generator=gen, device=device).mul_(3e-4).add_(1e-4).to(torch.float16)
    bias = torch.rand((R,), generator=gen, device=device).mul_(0.04).sub_(0.06).to(torch.float16)
    rows[:, D : D + 2] = scale.view(torch.uint8).view(R, 2)
    rows[:, D + 2 : D + 4] = bias.view(torch.uint8).view(R, 2)
    if stride > D + 4:
        rows[:, D + 4 :] = 0
    return rows


def _values_int8_rowwise_split(R, D, gen, device, stride):
    """The values of _values_int8_rowwise (same draws in the same order), in
    the split layout: rows of `stride` bytes holding the codes (zero padded),
    then the rows' (scale, bias) words.  Returns (rows view, storage)."""
    storage = torch.zeros((R * stride + 4 * R,), dtype=torch.uint8, device=device)
    rows = storage[:R * stride].view(R, stride)
    rows[:, :D] = torch.randint(0, 256, (R, D), generator=gen, device=device, dtype=torch.uint8)
    scale = torch.rand((R,), generator=gen, device=device).mul_(3e-4).add_(1e-4).to(torch.float16)
    bias = torch.rand((R,), generator=gen, device=device).mul_(0.04).sub_(0.06).to(torch.float16)
    words = storage[R * stride:].view(R, 4)
    words[:, 0:2] = scale.view(torch.uint8).view(R, 2)
    words[:, 2:4] = bias.view(torch.uint8).view(R, 2)
    return rows, storage


# ----------------------------------------------------------------------------
# bag-length laws (each returns int64 [B] on `device`)


def _len_uniform(lo, hi):
    def f(B, gen, device):
        return torch.randint(lo, hi + 1, (B,), generator=gen, device=device, dtype=torch.int64)

    return f


def _len_poisson(mean, cap):
    def f(B, gen, device):
        lam = torch.full((B,), float(mean), device=device, dtype=torch.float32)
        return torch.poisson(lam, generator=gen).to(torch.int64).clamp_(max=cap)

    return f


def _len_powerlaw(alpha, kmax):
    """P(k) proportional to k^-alpha on k = 1..kmax."""

    def f(B, gen, device):
        k = torch.arange(1, kmax + 1, device=device, dtype=torch.float64)
        cdf = k.pow(-alpha).cumsum(0)
        u = torch.rand((B,), generator=gen, device=device, dtype=torch.float64) * cdf[-1]
        return torch.searchsorted(cdf, u).clamp_(max=kmax - 1).add_(1).to(torch.int64)

    return f


def _len_one_hot():
    def f(B, gen, device):
        return torch.ones((B,), device=device, dtype=torch.int64)

    return f


def _len_geometric(p, cap):
    """Geometric on {1, 2, ...} with success probability p (mean 1/p), capped."""

    def f(B, gen, device):
        v = torch.empty((B,), device=device, dtype=torch.float64).geometric_(p, generator=gen)
        return v.to(torch.int64).clamp_(1, cap)

    return f


def _len_lognormal(mu, sigma, cap):
    def f(B, gen, device):
        v = torch.empty((B,), device=device, dtype=torch.float64).log_normal_(mu, sigma, generator=gen)
        return torch.round(v).clamp_(0, cap).to(torch.int64)

    return f


# ----------------------------------------------------------------------------
# index laws


def _coprime_multiplier(R: int, rng: np.random.Generator) -> int:
    if R == 1:
        return 1
    while True:
        a = int(rng.integers(1, R))
        if math.gcd(a, R) == 1:
            return a


def _indices(law, alpha, R, n, gen, rng, device):
    if n == 0:
        return torch.empty((0,), dtype=torch.int64, device=device)
    if law == "uniform":
        return torch.randint(0, R, (n,), generator=gen, device=device, dtype=torch.int64)
    # bounded Zipf over ranks 1..R, P(k) ~ k^-alpha, drawn by inverse CDF; the
    # rank -> row map is a seeded affine bijection so hot rows are scattered
    cdf = torch.arange(1, R + 1, device=device, dtype=torch.float64).pow_(-alpha).cumsum_(0)
    u = torch.rand((n,), generator=gen, device=device, dtype=torch.float64).mul_(cdf[-1])
    rank = torch.searchsorted(cdf, u).clamp_(max=R - 1)
    del cdf, u
    a = _coprime_multiplier(R, rng)
    c = int(rng.integers(0, R))
    return rank.mul_(a).add_(c).remainder_(R)


# ----------------------------------------------------------------------------
# the five workloads


@dataclass
class TableSpec:
    rows: int
    dim: int
    dtype: str
    values: str  # "uniform" | "normal" | "int8"
    lengths: Callable
    index_law: str  # "uniform" | "zipf"
    alpha: float = 0.0
    stride: Optional[int] = None  # int8 row stride in bytes


@dataclass
class ConfigSpec:
    name: str
    key: int
    batch: int
    pooling: str
    weighted: bool
    tables: Callable[[], List[TableSpec]]
    summary: str
    int8_layout: str = "packed"  # layout of int8 row-wise tables unless make_workload names one


def _c1_tables():
    return [TableSpec(1000, 16, F32, "uniform", _len_uniform(0, 8), "uniform")]


def _c2_tables():
    return [TableSpec(100_000, 64, F32, "normal", _len_poisson(20, 100), "zipf", 1.05) for _ in range(26)]


def _c3_tables():
    return [TableSpec(10_000_000, 128, F16, "normal", _len_powerlaw(1.2, 200), "zipf", 1.1) for _ in range(8)]


def _c4_tables():
    rng = _np_rng(4, 0, _S_PARAMS)
    one_hot = set(rng.permutation(100)[:40].tolist())
    specs = []
    for t in range(100):
        dim = int(rng.choice([32, 64, 128, 256]))
        rows = int(round(math.exp(rng.uniform(math.log(1e3), math.log(5e6)))))
        law = _len_one_hot() if t in one_hot else _len_geometric(1.0 / 30.0, 500)
        specs.append(TableSpec(rows, dim, F16, "normal", law, "zipf", 1.05))
    return specs


def _c5_tables():
    return [
        TableSpec(6_000_000, 128, INT8_ROWWISE, "int8", _len_lognormal(3.0, 1.0, 1000), "zipf", 1.05, stride=132)
        for _ in range(64)
    ]


CONFIGS = {
    "c1": ConfigSpec("c1", 1, 64, "sum", False, _c1_tables,
                     "1 fp32 table 1000x16 U(-1,1), B=64, lengths U{0..8}, uniform indices, sum"),
    "c2": ConfigSpec("c2", 2, 2048, "sum", False, _c2_tables,
                     "26 fp32 tables 100000x64 N(0,0.01), B=2048, Poisson(20) cap 100, Zipf 1.05, sum"),
    "c3a": ConfigSpec("c3a", 3, 16384, "mean", False, _c3_tables,
                      "8 fp16 tables 10Mx128 N(0,0.01), B=16384, power-law 1.2 on 1..200, Zipf 1.1, mean"),
    "c3b": ConfigSpec("c3b", 3, 16384, "sum", True, _c3_tables,
                      "8 fp16 tables 10Mx128 N(0,0.01), B=16384, power-law 1.2 on 1..200, Zipf 1.1, "
                      "weighted sum w~U(0,1)"),
    "c4": ConfigSpec("c4", 4, 8192, "sum", False, _c4_tables,
                     "100 fp16 tables D in {32,64,128,256}, rows log-U(1e3,5e6), B=8192, 40 one-hot + 60 "
                     "geometric(mean 30) cap 500, Zipf 1.05, sum"),
    # int8 rows in the split layout by default: on MI355X it was 3% faster than
    # the packed 132-byte rows under Zipf indices and 8% under uniform ones
    "c5": ConfigSpec("c5", 5, 65536, "sum", False, _c5_tables,
                     "64 int8-rowwise tables 6Mx128 (u8 codes + fp16 scale/bias per row, 50.7 GB), B=65536, "
                     "lognormal(3,1) cap 1000, Zipf 1.05, sum", int8_layout="split"),
}


def make_workload(
    name: str,
    device="cpu",
    *,
    batch_seed: int = 0,
    rows_cap: Optional[int] = None,
    batch: Optional[int] = None,
    num_tables: Optional[int] = None,
    index_dtype=torch.int64,
    index_law: Optional[str] = None,
    tables: Optional[List[Table]] = None,
    int8_layout: Optional[str] = None,
) -> Workload:
    """Draw one batch of config `name`.

    rows_cap / batch / num_tables shrink the shape (same laws) for tests that
    the oracle must finish in seconds; index_law="uniform" gives the
    no-reuse control; `tables` reuses tables drawn earlier (a new batch over
    the same tables: only lengths, indices and weights are drawn);
    int8_layout ("packed" or "split") stores int8 row-wise tables in that
    layout (default: the config's), with the same values either way.
    """
    cfg = CONFIGS[name]
    device = torch.device(device)
    specs = cfg.tables()
    if num_tables is not None:
        specs = specs[:num_tables]
    B = cfg.batch if batch is None else int(batch)
    k = cfg.key

    if tables is None:
        tables = []
        for t, s in enumerate(specs):
            R = s.rows if rows_cap is None else min(s.rows, rows_cap)
            gen = _torch_gen(device, k, t, _S_VALUES)
            if s.values == "uniform":
                rows = _values_uniform_f32(R, s.dim, gen, device)
            elif s.values == "normal":
                rows = _values_normal(R, s.dim, gen, device, torch.float32 if s.dtype == F32 else torch.float16)
            else:
                layout = int8_layout or cfg.int8_layout
                if layout not in INT8_LAYOUTS:
                    raise ValueError(f"int8_layout must be one of {sorted(INT8_LAYOUTS)}, got {layout!r}")
                if layout == "split":
                    stride = (s.dim + 15) // 16 * 16
                    rows, storage = _values_int8_rowwise_split(R, s.dim, gen, device, stride)
                    tables.append(Table(rows, s.dim, INT8_ROWWISE_SPLIT, storage))
                    continue
                rows = _values_int8_rowwise(R, s.dim, gen, device, s.stride or s.dim + 4)
            tables.append(Table(rows, s.dim, s.dtype))
    assert len(tables) == len(specs)

    lengths = torch.empty((len(specs), B), dtype=torch.int64, device=device)
    for t, s in enumerate(specs):
        lengths[t] = s.lengths(B, _torch_gen(device, k, t, _S_LENGTHS, batch_seed), device)
    lengths = lengths.reshape(-1)
    offsets = torch.zeros((lengths.numel() + 1,), dtype=torch.int64, device=device)
    torch.cumsum(lengths, 0, out=offsets[1:])
    n_total = int(offsets[-1].item())

    per_table = lengths.view(len(specs), B).sum(dim=1).cpu().tolist()
    indices = torch.empty((n_total,), dtype=torch.int64, device=device)
    pos = 0
    for t, s in enumerate(specs):
        n = int(per_table[t])
        law = index_law or s.index_law
        gen = _torch_gen(device, k, t, _S_INDICES, batch_seed)
        rng = _np_rng(k, t, _S_INDICES, batch_seed)
        indices[pos : pos + n] = _indices(law, s.alpha, tables[t].num_rows, n, gen, rng, device)
        pos += n

    weights = None
    if cfg.weighted:
        weights = torch.rand((n_total,), generator=_torch_gen(device, k, 0, _S_WEIGHTS, batch_seed),
                             device=device, dtype=torch.float32)

    if index_dtype != torch.int64:
        indices = indices.to(index_dtype)
        offsets = offsets.to(index_dtype)
    return Workload(name, tables, B, indices, offsets, weights, cfg.pooling, lengths)
