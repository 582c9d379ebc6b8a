"""GPU parity on tables larger than 4 GiB, through the C ABI.

Rows whose byte offset lies past 2^32 must be gathered (pooled and un-pooled
lookup) and updated (backward with row-wise Adagrad) exactly like low rows.
Two tables:
  * fp32, D = 128 (512-byte rows), 8.5 M rows (4.35 GB): rows from 8,388,608
    on start at or past 2^32;
  * int8 row-wise, D = 128 at the packed 132-byte stride, 32.6 M rows
    (4.30 GB): row 32,537,631 straddles 2^32 (its codes before, its scale
    and bias after);
  * int8 row-wise in the split layout, D = 128 at a 128-byte stride, 33.6 M
    rows (4.43 GB): rows from 33,554,432 on start at or past 2^32, and the
    whole scale/bias block lies past it.
Indices concentrate on the rows past the boundary, with the straddling row,
the last row and some low rows mixed in.  For the lookups the oracle runs on
the referenced rows only (a compact host copy with the indices renumbered
into it), which gives the same pooled values and sequence rows; the backward
is checked on the whole fp32 table.
"""
import numpy as np
import pytest
import torch

from conftest import compact_oracle_table
from oracle import OracleTable, ebo_forward, ebo_forward_seq
from paper_2609_30656_amd import eb
from paper_2609_30656_amd.workload import Workload
from test_backward_gpu import run_and_check
from test_parity_gpu import RTOL, _table, check, int8_parts, is_int8, per_element_lengths

pytestmark = pytest.mark.gpu

R_F32 = 8_500_000
R_U8 = 32_600_000
R_U8S = 33_600_000
FIRST_HIGH_F32 = 2 ** 32 // 512  # first fp32 row at or past 2^32
STRADDLE_U8 = 2 ** 32 // 132     # the int8 row that straddles 2^32
FIRST_HIGH_U8S = 2 ** 32 // 128  # first split-layout int8 row at or past 2^32
B = 384


def say(msg):
    print(msg, flush=True)


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    eb.load_library()
    d = torch.device("cuda:0")
    torch.cuda.set_device(d)
    return d


@pytest.fixture(scope="module")
def tables(dev):
    say(f"[large] generating tables: f32 {R_F32} x 128, int8 {R_U8} x 128 (stride 132), "
        f"split int8 {R_U8S} x 128 (stride 128)")
    t = [_table(dev, "f32", R_F32, 128, seed=41), _table(dev, "int8_rowwise", R_U8, 128, seed=42),
         _table(dev, "int8_rowwise_split", R_U8S, 128, seed=43)]
    assert t[0].rows.numel() * 4 > 2 ** 32 and t[1].rows.numel() > 2 ** 32 and t[2].rows.numel() > 2 ** 32
    assert 132 * STRADDLE_U8 < 2 ** 32 < 132 * (STRADDLE_U8 + 1)
    yield t
    del t
    torch.cuda.empty_cache()


def _indices(R, first_high, special, n, rng):
    """n row ids: 80% past the 4 GiB boundary, 20% anywhere, with the
    special rows placed first."""
    hi = rng.integers(first_high, R, n)
    lo = rng.integers(0, R, n)
    idx = np.where(rng.random(n) < 0.8, hi, lo)
    k = min(len(special), n)
    idx[:k] = special[:k]
    return idx


def _workload(dev, tables, weighted=False, pooling="sum", seed=0):
    rng = np.random.default_rng([2609, 99, seed])
    lens = [rng.integers(0, 25, B) for _ in tables]
    for L in lens:
        L[:4] = [1, 0, 1, 24]  # one-row, empty and long bags among the first
    idx = []
    for tb, L in zip(tables, lens):
        R = tb.num_rows
        if tb.dtype == "f32":
            special = [FIRST_HIGH_F32, FIRST_HIGH_F32 - 1, R - 1, 0]
        elif tb.dtype == "int8_rowwise":
            special = [STRADDLE_U8, STRADDLE_U8 - 1, STRADDLE_U8 + 1, R - 1]
        else:
            special = [FIRST_HIGH_U8S, FIRST_HIGH_U8S - 1, R - 1, 0]
        first_high = {"f32": FIRST_HIGH_F32, "int8_rowwise": STRADDLE_U8}.get(tb.dtype, FIRST_HIGH_U8S)
        idx.append(_indices(R, first_high, np.array(special), int(L.sum()), rng))
    lengths = torch.tensor(np.concatenate(lens), dtype=torch.int64)
    offsets = torch.zeros(lengths.numel() + 1, dtype=torch.int64)
    torch.cumsum(lengths, 0, out=offsets[1:])
    indices = torch.tensor(np.concatenate(idx), dtype=torch.int64)
    weights = torch.tensor(rng.random(indices.numel()), dtype=torch.float32) if weighted else None
    return Workload("large", list(tables), B, indices.to(dev), offsets.to(dev),
                    None if weights is None else weights.to(dev), pooling, lengths.to(dev))


def _compact(w):
    """Host copies of the referenced rows of each table, and the indices
    renumbered into them."""
    off = w.offsets.cpu().numpy()
    idx = w.indices.cpu().numpy()
    new = np.empty_like(idx)
    tabs = []
    for t, tb in enumerate(w.tables):
        lo, hi = int(off[t * w.batch]), int(off[(t + 1) * w.batch])
        u, inv = np.unique(idx[lo:hi], return_inverse=True)
        tabs.append(compact_oracle_table(tb, u))
        new[lo:hi] = inv
    return tabs, new, off


@pytest.mark.parametrize("mode", ["sum", "mean", "weighted"])
def test_pooled_lookup_past_4gib(dev, tables, mode):
    w = _workload(dev, tables, weighted=mode == "weighted", pooling="mean" if mode == "mean" else "sum")
    say(f"[large] pooled {mode}: {w.num_indices} lookups")
    out = torch.full((w.batch, w.sum_dim), float("nan"), device=dev)
    with eb.eb_create_tables(w.tables) as h:
        eb.eb_forward(h, w.indices, w.offsets, w.weights, w.pooling, out)
        torch.cuda.synchronize()
    tabs, idx, off = _compact(w)
    wts = None if w.weights is None else w.weights.cpu().numpy()
    ref, asum = ebo_forward(tabs, idx, off, wts, w.pooling, with_absum=True)
    got = out.cpu().numpy()
    L = per_element_lengths(w)
    D = 128
    for t, tb in enumerate(w.tables):
        cols = slice(t * D, (t + 1) * D)
        bscale = None
        if is_int8(tb.dtype) and mode != "weighted":
            # int8 rows sum s*q and the biases separately when unweighted: the
            # bound scale s' = sum(|s q|) + sum(|c|), the oracle's fp64
            # absolute sums over a table of |s| q and one of |c| in every
            # column (both exact in fp32)
            q, sc, bi = int8_parts(tabs[t])
            R = q.shape[0]
            prod = OracleTable(np.ascontiguousarray(q.astype(np.float32) * sc), D, "f32")
            bias = OracleTable(np.ascontiguousarray(np.broadcast_to(bi, (R, D))), D, "f32")
            others = [tabs[s] if s != t else None for s in range(len(tabs))]
            bscale = (ebo_forward([prod if x is None else x for x in others], idx, off, None, w.pooling,
                                  with_absum=True)[1][:, cols] +
                      ebo_forward([bias if x is None else x for x in others], idx, off, None, w.pooling,
                                  with_absum=True)[1][:, cols])
        check(got[:, cols], ref[:, cols], asum[:, cols], L[:, cols], RTOL[tb.dtype], f"large {tb.dtype} {mode}",
              bscale)


def test_sequence_lookup_past_4gib(dev, tables):
    w = _workload(dev, tables, seed=1)
    say(f"[large] sequence lookup: {w.num_indices} lookups")
    out = torch.full((w.num_indices * 128,), float("nan"), device=dev)
    with eb.eb_create_tables(w.tables) as h:
        eb.eb_forward_seq(h, w.indices, w.offsets, out)
        torch.cuda.synchronize()
    tabs, idx, off = _compact(w)
    ref = ebo_forward_seq(tabs, idx, off)
    got = out.cpu().numpy()
    same = got.view(np.uint32) == ref.view(np.uint32)
    assert same.all(), f"{np.count_nonzero(~same)} of {same.size} elements differ"


def test_backward_update_past_4gib(dev, tables):
    w = _workload(dev, tables[:1], seed=2)
    run_and_check(w, dev, "rowwise_adagrad", label="large f32")
