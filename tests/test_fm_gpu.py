"""GPU parity of the FM cross term (eb_fm_cross, and eb_forward_fm = lookup
then FM pass) against the oracle, through the C ABI.

Bar:
  * eb_forward_fm's out is bit-identical to eb_forward's out on the same
    inputs (the same kernel), so the forward's parity tests hold for it;
  * fm: |y_gpu - y_oracle| <= (rtol + c * 2^-24) * M with
    M = sum_d (sum_f A_{f,d})^2, A the oracle's per-element error scale of the
    pooled values, rtol the pooled bar (1e-5 fp32, 2e-3 fp16 / int8 row-wise)
    and c = 2T + 2 ceil(D / 64) + 16.  Pooled values within rtol * A move y
    by at most rtol (1 + rtol) M; evaluating 1/2 sum_d [(sum_f e)^2 - sum_f e^2]
    in fp32 adds at most c * 2^-24 * M (sums of T terms, the square and the
    difference, ceil(D/64) columns per lane, a 6-level butterfly, the half);
  * eb_fm_cross on a given fp32 matrix: the evaluation term alone,
    c * 2^-24 * sum_d (sum_f |e_{f,d}|)^2;
  * one field gives exactly +0.0.
"""
import numpy as np
import pytest
import torch

from conftest import compact_oracle_table
from oracle import OracleTable, ebo_fm, ebo_forward
from paper_2609_30656_amd import eb
from paper_2609_30656_amd.workload import make_workload
from test_parity_gpu import REDUCED, RTOL, _custom, _table

pytestmark = pytest.mark.gpu

U = 2.0 ** -24


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    eb.load_library()
    d = torch.device("cuda:0")
    torch.cuda.set_device(d)
    return d


def say(msg):
    print(msg, flush=True)


def run_fm(w, nan_fill=True):
    """eb_forward_fm and eb_forward on the same handle; returns (out_fm, fm, out_fwd)."""
    fill = float("nan") if nan_fill else 0.0
    out = torch.full((w.batch, w.sum_dim), fill, dtype=torch.float32, device=w.indices.device)
    ref = torch.full_like(out, fill)
    fm = torch.full((w.batch,), fill, dtype=torch.float32, device=w.indices.device)
    with eb.eb_create_tables(w.tables) as h:
        eb.eb_forward_fm(h, w.indices, w.offsets, w.weights, w.pooling, out, fm)
        eb.eb_forward(h, w.indices, w.offsets, w.weights, w.pooling, ref)
        torch.cuda.synchronize()
    return out, fm, ref


def sub_workload(w, examples):
    """The oracle's inputs for the listed examples only: their bags in the
    same table-major layout, each table cut down to the rows those bags read
    (renumbered).  Only data movement: no arithmetic of the method."""
    examples = np.asarray(examples, np.int64)
    B, T = w.batch, w.num_tables
    off = w.offsets.cpu().numpy().astype(np.int64)
    idx = w.indices.cpu().numpy().astype(np.int64)
    wts = None if w.weights is None else w.weights.cpu().numpy()
    tabs, new_idx, new_w, lens = [], [], [], []
    for t, tb in enumerate(w.tables):
        spans = [(off[t * B + b], off[t * B + b + 1]) for b in examples]
        pos = np.concatenate([np.arange(lo, hi) for lo, hi in spans]) if spans else np.zeros(0, np.int64)
        rows, inv = np.unique(idx[pos], return_inverse=True)
        tabs.append(compact_oracle_table(tb, rows))
        new_idx.append(inv.astype(np.int64))
        if wts is not None:
            new_w.append(wts[pos])
        lens += [hi - lo for lo, hi in spans]
    offsets = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    indices = np.concatenate(new_idx) if new_idx else np.zeros(0, np.int64)
    weights = np.concatenate(new_w).astype(np.float32) if wts is not None else None
    return tabs, indices, offsets, weights


def oracle_fm(w, examples=None):
    """Oracle pooled output, fm term and its error scale for the examples."""
    examples = np.arange(w.batch) if examples is None else np.asarray(examples)
    tabs, idx, off, wts = sub_workload(w, examples)
    pooled, asum = ebo_forward(tabs, idx, off, wts, w.pooling, with_absum=True)
    T, D = w.num_tables, w.tables[0].dim
    y, scale = ebo_fm(pooled, T, D, asum)
    return pooled, y, scale


def check_fm(got_fm, y, scale, w, label):
    got = np.asarray(got_fm, np.float32).astype(np.float64)
    assert not np.isnan(got).any(), f"{label}: fm element not written"
    T, D = w.num_tables, w.tables[0].dim
    rtol = RTOL[w.tables[0].dtype]
    c = 2 * T + 2 * -(-D // 64) + 16
    lim = (rtol + c * U) * scale
    err = np.abs(got - y)
    bad = err > lim
    assert not bad.any(), (f"{label}: {bad.sum()} fm values beyond the bound; worst ratio "
                           f"{np.max(err / np.maximum(lim, 1e-300)):.3g}")


def full_fm_check(w, label):
    out, fm, ref = run_fm(w)
    assert torch.equal(out.view(torch.int32), ref.view(torch.int32)), f"{label}: out differs from eb_forward"
    _, y, scale = oracle_fm(w)
    check_fm(fm.cpu().numpy(), y, scale, w, label)
    return fm


FM_CONFIGS = ["c1", "c2", "c3a", "c3b", "c5"]  # every table of one width and storage type


@pytest.mark.parametrize("name", FM_CONFIGS)
def test_reduced_configs(dev, name):
    say(f"[fm] reduced {name} {REDUCED[name]}")
    w = make_workload(name, dev, **REDUCED[name])
    fm = full_fm_check(w, f"reduced {name}")
    if w.num_tables == 1:
        assert torch.equal(fm.view(torch.int32), torch.zeros_like(fm).view(torch.int32))


@pytest.mark.parametrize("name", ["c3a", "c5"])
def test_with_the_long_bag_pass(dev, monkeypatch, name):
    # most bags pooled by the long-bag pass (EB_LONG_BAG=16, segments of 64):
    # eb_forward_fm's pooled output is still eb_forward's, bit for bit, and
    # the term holds the oracle's bound
    say(f"[fm] long-bag pass {name}")
    monkeypatch.setenv("EB_LONG_BAG", "16")
    monkeypatch.setenv("EB_LONG_SEG", "64")
    w = make_workload(name, dev, **REDUCED[name])
    full_fm_check(w, f"long-bag pass {name}")


@pytest.mark.parametrize("name", ["c2", "c5"])
def test_int32_indices(dev, name):
    say(f"[fm] int32 {name}")
    w = make_workload(name, dev, index_dtype=torch.int32, **REDUCED[name])
    full_fm_check(w, f"int32 {name}")


def _fm_pass_check(dev, T, D, B, seed, scale=1.0):
    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    e = torch.randn((B, T * D), generator=g, device=dev) * scale
    tables = [_table(dev, "f32", 4, D, seed=t) for t in range(T)]
    fm = torch.full((B,), float("nan"), device=dev)
    with eb.eb_create_tables(tables) as h:
        eb.eb_fm_cross(h, e, fm)
        torch.cuda.synchronize()
    host = e.cpu().numpy()
    y = ebo_fm(host, T, D)
    M = (np.abs(host.astype(np.float64)).reshape(B, T, D).sum(axis=1) ** 2).sum(axis=1)
    c = 2 * T + 2 * -(-D // 64) + 16
    err = np.abs(fm.cpu().numpy().astype(np.float64) - y)
    assert np.all(err <= c * U * M), f"T={T} D={D}: worst {np.max(err / (c * U * M)):.3g} of the bound"
    return fm


@pytest.mark.parametrize("T,D", [(1, 64), (2, 4), (3, 12), (26, 64), (8, 128), (64, 128), (5, 256), (4, 260),
                                 (3, 1028), (70, 8), (300, 16)])
def test_fm_pass_alone(dev, T, D):
    say(f"[fm] eb_fm_cross T={T} D={D}")
    fm = _fm_pass_check(dev, T, D, 75, seed=T * 1000 + D)
    if T == 1:
        assert torch.equal(fm.view(torch.int32), torch.zeros_like(fm).view(torch.int32))


def test_fm_pass_argument_errors(dev):
    say("[fm] eb_fm_cross argument errors")
    tables = [_table(dev, "f32", 4, 8, seed=t) for t in range(3)]
    with eb.eb_create_tables(tables) as h:
        for pooled, fm, status in [
                (torch.zeros(5 * 24 + 8, device=dev), torch.zeros(5, device=dev), eb.EB_ERR_SHAPE),
                (torch.zeros(5 * 24, device=dev), torch.zeros(4, device=dev), eb.EB_ERR_SHAPE),
                (torch.zeros(5 * 24, device=dev, dtype=torch.int32), torch.zeros(5, device=dev), eb.EB_ERR_DTYPE),
                (torch.zeros(5 * 24, device=dev), None, eb.EB_ERR_INVALID_ARG),
                (torch.zeros(5 * 24 + 1, device=dev)[1:], torch.zeros(5, device=dev), eb.EB_ERR_UNSUPPORTED)]:
            with pytest.raises(eb.EBError) as e:
                eb.eb_fm_cross(h, pooled, fm)
            assert e.value.status == status
    with eb.eb_create_tables([_table(dev, "f32", 4, 8), _table(dev, "f32", 4, 16)]) as h:
        with pytest.raises(eb.EBError) as e:
            eb.eb_fm_cross(h, torch.zeros(24, device=dev), torch.zeros(1, device=dev))
        assert e.value.status == eb.EB_ERR_SHAPE


FM_WIDTHS = [("f32", 4), ("f32", 12), ("f32", 64), ("f32", 256), ("f32", 260), ("f32", 1028),
             ("f16", 8), ("f16", 24), ("f16", 128), ("f16", 520),
             ("int8_rowwise", 16), ("int8_rowwise", 48), ("int8_rowwise", 128), ("int8_rowwise", 2064),
             ("int8_rowwise_split", 128), ("int8_rowwise_split", 2064)]


@pytest.mark.parametrize("mode", ["sum", "mean", "weighted"])
@pytest.mark.parametrize("dtype,D", FM_WIDTHS)
def test_every_kind(dev, dtype, D, mode):
    say(f"[fm] kind {dtype} D{D} {mode}")
    rng = np.random.default_rng(D)
    T, B = 5, 37
    tables = [_table(dev, dtype, 200 + 13 * t, D, seed=t) for t in range(T)]
    lens = [rng.integers(0, 80, B) for _ in tables]
    for l in lens:
        l[0], l[1], l[2] = 0, 1, 70  # empty, one row, past one index chunk
    w = _custom(dev, tables, lens, weighted=(mode == "weighted"), pooling="mean" if mode == "mean" else "sum")
    full_fm_check(w, f"{dtype} D{D} {mode}")


@pytest.mark.parametrize("T", [1, 2, 3, 7, 261])
def test_table_counts(dev, T):
    # fewer tables than waves (idle waves), and more than 64 tables per wave
    say(f"[fm] T={T}")
    rng = np.random.default_rng(T)
    B = 9
    tables = [_table(dev, "f32", 60, 8, seed=t) for t in range(T)]
    w = _custom(dev, tables, [rng.integers(0, 20, B) for _ in tables])
    fm = full_fm_check(w, f"T={T}")
    if T == 1:
        assert torch.equal(fm.view(torch.int32), torch.zeros_like(fm).view(torch.int32))


def test_no_indices_at_all(dev):
    say("[fm] N = 0")
    tables = [_table(dev, "f16", 50, 64, seed=t) for t in range(4)]
    w = _custom(dev, tables, [np.zeros(6, np.int64) for _ in tables])
    out, fm, _ = run_fm(w)
    assert torch.equal(out.view(torch.int32), torch.zeros_like(out).view(torch.int32))
    assert torch.equal(fm.view(torch.int32), torch.zeros_like(fm).view(torch.int32))


def test_deterministic_bits(dev):
    say("[fm] determinism")
    w = make_workload("c5", dev, **REDUCED["c5"])
    o1, f1, _ = run_fm(w)
    o2, f2, _ = run_fm(w)
    assert torch.equal(o1.view(torch.int32), o2.view(torch.int32))
    assert torch.equal(f1.view(torch.int32), f2.view(torch.int32))


def test_full_c2_every_example(dev):
    say("[fm] full c2")
    full_fm_check(make_workload("c2", dev), "full c2")


@pytest.mark.parametrize("name", ["c3a", "c3b", "c5", "c5-packed"])
def test_full_size_sampled(dev, name):
    say(f"[fm] full {name}: generating")
    name, _, layout = name.partition("-")
    w = make_workload(name, dev, int8_layout=layout or None)
    say(f"[fm] full {name}: {w.num_indices} lookups; forward_fm")
    out, fm, ref = run_fm(w)
    assert torch.equal(out.view(torch.int32), ref.view(torch.int32))
    assert not torch.isnan(fm).any()
    lens = w.lengths.view(w.num_tables, w.batch).sum(0).cpu().numpy()
    rng = np.random.default_rng(1)
    ex = np.unique(np.concatenate([[0, w.batch - 1, int(np.argmax(lens)), int(np.argmin(lens))],
                                   rng.choice(w.batch, 60, replace=False)]))
    say(f"[fm] full {name}: oracle on {ex.size} examples")
    pooled, y, scale = oracle_fm(w, ex)
    check_fm(fm.cpu().numpy()[ex], y, scale, w, f"full {name}")


def test_argument_errors(dev):
    say("[fm] argument errors")
    w = make_workload("c2", dev, rows_cap=1000, batch=8, num_tables=3)
    out = torch.empty((w.batch, w.sum_dim), device=dev)
    fm = torch.empty(w.batch, device=dev)
    with eb.eb_create_tables(w.tables) as h:
        for bad, status in [(torch.empty(w.batch + 1, device=dev), eb.EB_ERR_SHAPE),
                            (torch.empty(w.batch, device=dev, dtype=torch.int32), eb.EB_ERR_DTYPE),
                            (None, eb.EB_ERR_INVALID_ARG)]:
            with pytest.raises(eb.EBError) as e:
                eb.eb_forward_fm(h, w.indices, w.offsets, w.weights, w.pooling, out, bad)
            assert e.value.status == status
        with pytest.raises(eb.EBError) as e:
            eb.eb_forward_fm(h, w.indices, w.offsets, torch.ones(w.num_indices, device=dev), "mean", out, fm)
        assert e.value.status == eb.EB_ERR_INVALID_ARG
    mixed_dim = [_table(dev, "f32", 10, 8), _table(dev, "f32", 10, 16)]
    wk = _custom(dev, mixed_dim, [np.ones(3, np.int64) for _ in mixed_dim])
    o = torch.empty((3, wk.sum_dim), device=dev)
    with eb.eb_create_tables(wk.tables) as h:
        with pytest.raises(eb.EBError) as e:
            eb.eb_forward_fm(h, wk.indices, wk.offsets, None, "sum", o, torch.empty(3, device=dev))
        assert e.value.status == eb.EB_ERR_SHAPE


def test_mixed_storage_types_of_one_width(dev):
    say("[fm] fp32 + fp16 + int8 tables of one width")
    rng = np.random.default_rng(8)
    tables = [_table(dev, "f32", 90, 64, seed=0), _table(dev, "f16", 80, 64, seed=1),
              _table(dev, "int8_rowwise", 70, 64, seed=2), _table(dev, "f16", 60, 64, seed=3)]
    w = _custom(dev, tables, [rng.integers(0, 30, 21) for _ in tables], weighted=True)
    out, fm, ref = run_fm(w)
    assert torch.equal(out.view(torch.int32), ref.view(torch.int32))
    _, y, scale = oracle_fm(w)
    got = fm.cpu().numpy().astype(np.float64)
    c = 2 * len(tables) + 2 + 16
    assert np.all(np.abs(got - y) <= (2e-3 + c * U) * scale)


def test_checked_mode_reports_bad_index(dev, monkeypatch):
    say("[fm] checked mode")
    monkeypatch.setenv("EB_CHECK", "1")
    tables = [_table(dev, "f32", 40, 16, seed=t) for t in range(3)]
    w = _custom(dev, tables, [np.full(4, 2, np.int64) for _ in tables])
    w.indices[5] = 40  # one past the end of table 0
    out = torch.empty((4, w.sum_dim), device=dev)
    fm = torch.empty(4, device=dev)
    with eb.eb_create_tables(w.tables) as h:
        with pytest.raises(eb.EBError) as e:
            eb.eb_forward_fm(h, w.indices, w.offsets, None, "sum", out, fm)
        assert e.value.status == eb.EB_ERR_INDEX_OOB
