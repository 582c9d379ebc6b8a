"""The seeded generator draws the shapes and laws it claims (CPU only)."""
import numpy as np
import pytest
import torch

from paper_2609_30656_amd.workload import CONFIGS, make_workload


@pytest.mark.parametrize("name", list(CONFIGS))
def test_structure(name):
    w = make_workload(name, "cpu", rows_cap=3000, batch=128, num_tables=5)
    T, B = w.num_tables, w.batch
    off = w.offsets.numpy()
    assert off.shape == (T * B + 1,) and off[0] == 0 and off[-1] == w.num_indices
    assert np.all(np.diff(off) >= 0)
    assert np.array_equal(np.diff(off), w.lengths.numpy())
    idx = w.indices.numpy()
    for t, tab in enumerate(w.tables):
        seg = idx[off[t * B]:off[(t + 1) * B]]
        assert seg.size == 0 or (seg.min() >= 0 and seg.max() < tab.num_rows)
    if w.weights is not None:
        assert w.weights.shape == (w.num_indices,) and w.weights.min() >= 0 and w.weights.max() < 1


def test_deterministic_and_batch_seeds_differ():
    a = make_workload("c2", "cpu", rows_cap=2000, batch=64, num_tables=3)
    b = make_workload("c2", "cpu", rows_cap=2000, batch=64, num_tables=3)
    c = make_workload("c2", "cpu", rows_cap=2000, batch=64, num_tables=3, batch_seed=1, tables=a.tables)
    assert torch.equal(a.indices, b.indices) and torch.equal(a.tables[0].rows, b.tables[0].rows)
    assert not torch.equal(a.indices, c.indices) or not torch.equal(a.offsets, c.offsets)


def test_length_laws():
    c1 = make_workload("c1", "cpu", batch=20000).lengths.numpy()
    assert c1.min() == 0 and c1.max() == 8 and abs(c1.mean() - 4) < 0.1
    c2 = make_workload("c2", "cpu", rows_cap=100, batch=20000, num_tables=1).lengths.numpy()
    assert c2.max() <= 100 and abs(c2.mean() - 20) < 0.2
    c3 = make_workload("c3a", "cpu", rows_cap=100, batch=40000, num_tables=1).lengths.numpy()
    assert c3.min() >= 1 and c3.max() <= 200 and abs(c3.mean() - 22.3) < 1.0
    c5 = make_workload("c5", "cpu", rows_cap=100, batch=40000, num_tables=1).lengths.numpy()
    # lognormal(3, 1) rounded and capped at 1000: mean exp(3.5) ~ 33.1
    assert c5.max() <= 1000 and abs(c5.mean() - 33.1) < 1.5


def test_c4_mix():
    specs = CONFIGS["c4"].tables()
    dims = [s.dim for s in specs]
    rows = [s.rows for s in specs]
    assert set(dims) <= {32, 64, 128, 256} and len(set(dims)) == 4
    assert 1000 <= min(rows) and max(rows) <= 5_000_000
    w = make_workload("c4", "cpu", rows_cap=100, batch=4000)
    per = w.lengths.view(100, -1)
    one_hot = [(per[t] == 1).all().item() for t in range(100)]
    assert sum(one_hot) == 40
    jag = per[[t for t in range(100) if not one_hot[t]]].double()
    assert jag.min() >= 1 and jag.max() <= 500 and abs(jag.mean().item() - 30) < 1


def test_zipf_is_skewed_and_uniform_is_not():
    z = make_workload("c2", "cpu", batch=2048, num_tables=1).indices.numpy()
    u = make_workload("c2", "cpu", batch=2048, num_tables=1, index_law="uniform").indices.numpy()
    for arr, lo, hi in ((z, 0.5, 1.0), (u, 0.0, 0.1)):
        cnt = np.sort(np.bincount(arr, minlength=100_000))[::-1]
        top1 = cnt[:1000].sum() / arr.size  # share of lookups hitting the top 1% of rows
        assert lo <= top1 <= hi


def test_int8_row_layout():
    w = make_workload("c5", "cpu", rows_cap=500, batch=8, num_tables=2, int8_layout="packed")
    t = w.tables[0]
    assert t.dtype == "int8_rowwise"
    assert t.rows.dtype == torch.uint8 and t.row_stride_bytes == 132 and t.row_bytes == 132
    s = t.rows[:, 128:130].contiguous().view(torch.float16).float()
    c = t.rows[:, 130:132].contiguous().view(torch.float16).float()
    assert s.min() >= 0.99e-4 and s.max() <= 4.01e-4 and c.min() >= -0.0601 and c.max() <= -0.0199


def test_int8_split_layout_holds_the_packed_values():
    # c5's default layout: codes in 128-byte rows, then the scale/bias block;
    # the same draws as the packed layout, byte for byte
    split = make_workload("c5", "cpu", rows_cap=500, batch=8, num_tables=2)
    packed = make_workload("c5", "cpu", rows_cap=500, batch=8, num_tables=2, int8_layout="packed")
    for s, p in zip(split.tables, packed.tables):
        R = s.num_rows
        assert s.dtype == "int8_rowwise_split" and s.row_stride_bytes == 128 and s.row_bytes == 132
        assert s.storage.numel() == R * 132 and s.rows.data_ptr() == s.storage.data_ptr()
        assert torch.equal(s.rows[:, :128], p.rows[:, :128])
        assert torch.equal(s.storage[R * 128:].view(R, 4), p.rows[:, 128:132])
        assert s.host_bytes().shape == (R * 132,)
        c = s.clone()
        assert torch.equal(c.storage, s.storage) and c.storage.data_ptr() != s.storage.data_ptr()
    assert torch.equal(split.indices, packed.indices) and torch.equal(split.offsets, packed.offsets)
    assert split.algorithmic_bytes() == packed.algorithmic_bytes()


def test_algorithmic_bytes_counts_every_term():
    w = make_workload("c3b", "cpu", rows_cap=100, batch=16, num_tables=2)
    N = w.num_indices
    expect = N * 256 + N * 8 + (2 * 16 + 1) * 8 + N * 4 + 16 * 256 * 4
    assert w.algorithmic_bytes() == expect


def test_sequence_and_backward_byte_counts():
    from oracle import ebo_forward_seq
    from conftest import oracle_tables

    w = make_workload("c4", "cpu", rows_cap=300, batch=6, num_tables=5)
    seq = ebo_forward_seq(oracle_tables(w), w.indices.numpy(), w.offsets.numpy())
    assert w.seq_output_numel() == seq.size
    off, B, esz = w.offsets.numpy(), w.batch, w.indices.element_size()
    n = [int(off[(t + 1) * B] - off[t * B]) for t in range(w.num_tables)]
    assert w.table_lookups() == n
    expect = (w.num_tables + 1) * esz + sum(n[t] * (tb.row_bytes + esz + 4 * tb.dim) for t, tb in enumerate(w.tables))
    assert w.seq_algorithmic_bytes() == expect
    idx = w.indices.numpy()
    uniq = [np.unique(idx[off[t * B]:off[(t + 1) * B]]).size for t in range(w.num_tables)]
    expect = w.num_indices * esz + off.size * esz + sum(
        n[t] * 4 * tb.dim + uniq[t] * (2 * tb.row_bytes + 8) for t, tb in enumerate(w.tables))
    assert w.backward_algorithmic_bytes() == expect
