"""Pins for the oracle's un-pooled (sequence) lookup.

Every position's row as fp32, table t's positions forming a [N_t, D_t] block,
the blocks in table order.  Pinned by hand-worked cases, torch's CPU
embedding lookup, the pooled oracle (the fp64 sum of a bag's sequence rows,
rounded once, is the pooled sum bit for bit, and a one-row bag is its row),
and error codes.
"""
import numpy as np
import pytest
import torch

from conftest import oracle_forward, oracle_tables
from oracle import OracleError, OracleTable, ebo_forward_seq
from paper_2609_30656_amd.workload import make_workload

W4 = np.array([[1, 2], [3, 4], [5, 6], [7, 8]], dtype=np.float32)


def test_worked_one_and_two_tables():
    out = ebo_forward_seq([OracleTable(W4, 2, "f32")], np.array([2, 0, 3, 3]), np.array([0, 2, 2, 4]))
    np.testing.assert_array_equal(out, [5, 6, 1, 2, 7, 8, 7, 8])
    W3 = np.arange(9, dtype=np.float32).reshape(3, 3) * 10
    # T = 2, B = 2: table 0 bags {1}, {0, 3}; table 1 bags {2}, {}
    out = ebo_forward_seq([OracleTable(W4, 2, "f32"), OracleTable(W3, 3, "f32")],
                          np.array([1, 0, 3, 2]), np.array([0, 1, 3, 4, 4]))
    np.testing.assert_array_equal(out, [3, 4, 1, 2, 7, 8, 60, 70, 80])


def test_worked_int8_row():
    row = np.zeros((1, 6), np.uint8)
    row[0, 0], row[0, 1] = 0, 255
    row[0, 2:4] = np.frombuffer(np.float16(0.5).tobytes(), np.uint8)
    row[0, 4:6] = np.frombuffer(np.float16(-1.0).tobytes(), np.uint8)
    out = ebo_forward_seq([OracleTable(row, 2, "int8_rowwise")], np.array([0, 0]), np.array([0, 2]))
    np.testing.assert_array_equal(out, [-1, 126.5, -1, 126.5])


@pytest.mark.parametrize("name", ["c1", "c2", "c3a", "c4"])
def test_torch_embedding(name):
    w = make_workload(name, "cpu", rows_cap=500, batch=16, num_tables=4)
    tabs = oracle_tables(w)
    idx, off = w.indices.numpy(), w.offsets.numpy()
    out = ebo_forward_seq(tabs, idx, off)
    B, pos = w.batch, 0
    for t, tb in enumerate(w.tables):
        lo, hi = off[t * B], off[(t + 1) * B]
        ref = torch.nn.functional.embedding(torch.from_numpy(idx[lo:hi]), tb.rows.float()).numpy()
        n = ref.size
        assert np.array_equal(out[pos:pos + n].view(np.uint32), ref.reshape(-1).view(np.uint32))
        pos += n
    assert pos == out.size


@pytest.mark.parametrize("name", ["c2", "c3a", "c4", "c5"])
def test_bag_sums_are_the_pooled_lookup(name):
    w = make_workload(name, "cpu", rows_cap=400, batch=12, num_tables=3)
    tabs = oracle_tables(w)
    idx, off = w.indices.numpy(), w.offsets.numpy()
    seq = ebo_forward_seq(tabs, idx, off)
    pooled = oracle_forward(w, tables=tabs, with_absum=False)
    B, pos, col = w.batch, 0, 0
    for t, tb in enumerate(w.tables):
        D = tb.dim
        for b in range(B):
            g = t * B + b
            L = off[g + 1] - off[g]
            rows = seq[pos:pos + L * D].reshape(L, D).astype(np.float64)
            s = np.zeros(D)
            for r in rows:  # in index order, as the pooled oracle sums
                s = s + r
            expect = (s / L if (w.pooling == "mean" and L) else s).astype(np.float32)
            assert np.array_equal(pooled[b, col:col + D].view(np.uint32), expect.view(np.uint32)), (t, b)
            pos += L * D
        col += D
    assert pos == seq.size


def test_seq_error_codes():
    t = OracleTable(W4, 2, "f32")
    with pytest.raises(OracleError) as e:
        ebo_forward_seq([t], np.array([2, 0, 3, 3]), np.array([0, 2, 2, 4]), out_numel=7)
    assert e.value.code == -3
    with pytest.raises(OracleError) as e:
        ebo_forward_seq([t], np.array([2, 0, 4, 3]), np.array([0, 2, 2, 4]))
    assert e.value.code == -5
    with pytest.raises(OracleError) as e:
        ebo_forward_seq([t], np.array([2, 0, 3, 3]), np.array([0, 3, 2, 4]), out_numel=8)
    assert e.value.code == -6
