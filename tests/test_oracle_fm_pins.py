"""Pins for the oracle's factorization-machine cross term.

y_b = sum over unordered pairs of distinct fields f < f' of <e_{b,f}, e_{b,f'}>,
with e_{b,f} the pooled embedding of field (table) f for example b (the FM
second-order term over fields; Sec. IV-A.2 of the paper names the fm
submodule, the Introduction cites the factorization machine).  The oracle
sums the pairs directly.  It is pinned by hand-worked cases, the sum-of-squares
identity of the FM, the Gram-matrix form in torch, a brute force from the raw
table rows that never forms the pooled vectors, invariants, and error codes.
"""
import numpy as np
import pytest
import torch

from conftest import oracle_forward, oracle_tables
from oracle import OracleError, ebo_fm
from paper_2609_30656_amd.workload import make_workload


def test_worked_two_and_three_fields():
    assert ebo_fm(np.array([[1, 2, 3, 4]], np.float32), 2, 2)[0] == 11.0
    # [1,0], [0,1], [2,3]: pairs 0, 2, 3
    assert ebo_fm(np.array([[1, 0, 0, 1, 2, 3]], np.float32), 3, 2)[0] == 5.0
    # two examples, padding columns past T*D are ignored
    e = np.array([[1, 1, 1, 1, 99], [2, 0, -1, 5, -99]], np.float32)
    np.testing.assert_array_equal(ebo_fm(e, 2, 2), [2.0, -2.0])


def test_single_field_is_zero_and_identical_fields_give_the_squared_norm():
    rng = np.random.default_rng(11)
    e = rng.standard_normal((7, 16)).astype(np.float32)
    np.testing.assert_array_equal(ebo_fm(e, 1, 16), np.zeros(7))
    two = np.concatenate([e, e], axis=1)
    expect = (e.astype(np.float64) ** 2).sum(axis=1)
    np.testing.assert_allclose(ebo_fm(two, 2, 16), expect, rtol=1e-15)


def _identity(e, T, D):
    x = e[:, :T * D].astype(np.float64).reshape(-1, T, D)
    return 0.5 * ((x.sum(axis=1) ** 2) - (x ** 2).sum(axis=1)).sum(axis=1)


@pytest.mark.parametrize("T,D", [(2, 4), (5, 8), (26, 64), (3, 1)])
def test_sum_of_squares_identity(T, D):
    rng = np.random.default_rng(T * 100 + D)
    e = rng.standard_normal((33, T * D + 3)).astype(np.float32)
    y = ebo_fm(e, T, D)
    scale = (np.abs(e[:, :T * D].astype(np.float64)).reshape(-1, T, D).sum(axis=1) ** 2).sum(axis=1)
    assert np.all(np.abs(y - _identity(e, T, D)) <= 1e-13 * scale)


def test_gram_matrix_form_in_torch():
    rng = np.random.default_rng(12)
    T, D = 9, 24
    e = rng.standard_normal((20, T * D)).astype(np.float32)
    E = torch.from_numpy(e).double().reshape(20, T, D)
    G = torch.bmm(E, E.transpose(1, 2).contiguous())
    ref = torch.triu(G, diagonal=1).sum(dim=(1, 2)).numpy()
    np.testing.assert_allclose(ebo_fm(e, T, D), ref, rtol=1e-12, atol=1e-12)


def _row_values(table, rows):
    """fp64 element values of the given rows, from the storage format."""
    a = table.rows
    if table.dtype == "f32":
        return a[rows].astype(np.float64)
    if table.dtype == "f16":
        return a[rows].astype(np.float64)
    D = table.dim
    if table.dtype == "int8_rowwise_split":
        R, st = table.num_rows, table.row_stride
        buf = a.reshape(-1)
        codes = buf[:R * st].reshape(R, st)[rows, :D].astype(np.float64)
        sb = np.ascontiguousarray(buf[R * st:R * st + 4 * R].reshape(R, 4)[rows]).view(np.float16)
    else:
        codes = a[rows, :D].astype(np.float64)
        sb = np.ascontiguousarray(a[rows, D:D + 4]).view(np.float16)
    sb = sb.astype(np.float64)
    return (sb[:, :1] * codes + sb[:, 1:2]).astype(np.float32).astype(np.float64)


@pytest.mark.parametrize("name", ["c2", "c3a", "c3b", "c5", "c5-packed"])
def test_brute_force_from_table_rows(name):
    name, _, layout = name.partition("-")
    w = make_workload(name, "cpu", rows_cap=400, batch=12, num_tables=4, int8_layout=layout or None)
    tabs = oracle_tables(w)
    T, B, D = len(tabs), w.batch, tabs[0].dim
    pooled, asum = oracle_forward(w, tables=tabs)
    y, scale = ebo_fm(pooled, T, D, asum)
    idx, off = w.indices.numpy(), w.offsets.numpy()
    wt = None if w.weights is None else w.weights.numpy().astype(np.float64)
    for b in range(B):
        vecs, coefs = [], []
        for t in range(T):
            g = t * B + b
            lo, hi = off[g], off[g + 1]
            vecs.append(_row_values(tabs[t], idx[lo:hi]))
            if w.pooling == "mean":
                c = np.full(hi - lo, 1.0 / max(hi - lo, 1))
            else:
                c = np.ones(hi - lo) if wt is None else wt[lo:hi]
            coefs.append(c)
        ref = 0.0
        for f in range(T):
            for g2 in range(f + 1, T):
                # every pair of rows from two different fields, never pooling first
                ref += float(coefs[f] @ (vecs[f] @ vecs[g2].T) @ coefs[g2])
        # the oracle works from the pooled values rounded to fp32: each moves by
        # at most 2^-24 of its magnitude, so y moves by at most ~2^-23 * scale
        assert abs(y[b] - ref) <= 2.0 ** -22 * scale[b], (b, y[b], ref, scale[b])


def test_invariants_permutation_and_scaling():
    rng = np.random.default_rng(13)
    T, D = 6, 8
    e = rng.standard_normal((15, T * D)).astype(np.float32)
    y = ebo_fm(e, T, D)
    perm = rng.permutation(T)
    ep = e.reshape(15, T, D)[:, perm].reshape(15, T * D)
    scale = (np.abs(e.astype(np.float64)).reshape(15, T, D).sum(axis=1) ** 2).sum(axis=1)
    assert np.all(np.abs(ebo_fm(ep, T, D) - y) <= 1e-14 * scale)
    np.testing.assert_array_equal(ebo_fm(2 * e, T, D), 4 * y)  # powers of two are exact


def test_scale_bounds_the_term():
    w = make_workload("c3b", "cpu", rows_cap=300, batch=10, num_tables=3)
    pooled, asum = oracle_forward(w)
    T, D = 3, w.tables[0].dim
    y, scale = ebo_fm(pooled, T, D, asum)
    ref = (asum.reshape(w.batch, T, D).sum(axis=1) ** 2).sum(axis=1)
    np.testing.assert_allclose(scale, ref, rtol=1e-15)
    assert np.all(np.abs(y) <= 0.5 * scale * (1 + 2.0 ** -22))


def test_fm_error_codes():
    e = np.zeros((2, 6), np.float32)
    with pytest.raises(OracleError) as err:
        ebo_fm(e, 4, 2)  # 4 fields of 2 need 8 columns
    assert err.value.code == -3
    with pytest.raises(OracleError) as err:
        ebo_fm(e, 3, 0)
    assert err.value.code == -1
