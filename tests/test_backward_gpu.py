"""GPU parity of the backward + fused optimizer step against the CPU oracle.

For every table row the oracle reports (rows that occur in the batch) with
gradient G (fp64), error scale S = sum_i |c_i g| and occurrence count n:
  * rows that do not occur keep their bits;
  * SGD:    |W_gpu - W_oracle| <= lr (n + 8) u S + rounding of the stored value
            (2u|W| for fp32 tables, one fp16 ulp for fp16 tables);
  * Adagrad: the same with the error of the state and of the step size
            propagated (bounds computed below from G, S, n), and the state
            itself within its bound,
with u = 2^-24: fp32 summation of the n terms in any order, the tile partial
sums included.  Those bounds are first order in u: each term is k u X with
k <= n + 16.  Higham's gamma_k = k u / (1 - k u) makes such a term rigorous
(the roundings' second-order products included), and gamma_k <= k u / (1 -
(n + 16) u) for every such k, so the first-order bound divided by
1 - (n + 16) u is a rigorous one.  The Adagrad step size sigma = lr /
(sqrt(s) + eps) is taken with its exact perturbation: a state off by at most
ds moves sqrt(s) by at most ds / (sqrt(s) + sqrt(max(s - ds, 0))), so sigma
moves by at most that over (sqrt(max(s - ds, 0)) + eps) relative to itself,
for any ds; its own roundings add gamma_6.
"""
import numpy as np
import pytest
import torch

from oracle import OracleTable, ebo_backward_update
from paper_2609_30656_amd import eb
from paper_2609_30656_amd.workload import Table, Workload, make_workload

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


def _grad(w, dev, seed=7):
    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    return torch.randn((w.batch, w.sum_dim), generator=g, device=dev, dtype=torch.float32)


def _ulp16(x):
    """One fp16 ulp at |x| (subnormal spacing below 2^-14)."""
    a = np.maximum(np.abs(x), 2.0 ** -14)
    return 2.0 ** (np.floor(np.log2(a)) - 10)


def run_and_check(w, dev, optimizer, lr=0.05, eps=1e-4, check_tables=None, label=""):
    T = w.num_tables
    check_tables = list(range(T)) if check_tables is None else check_tables
    grad = _grad(w, dev)
    R = [t.num_rows for t in w.tables]
    state = None
    if optimizer == "rowwise_adagrad":
        gs = torch.Generator(device=dev)
        gs.manual_seed(11)
        state = torch.rand(sum(R), generator=gs, device=dev, dtype=torch.float32)
    before = {t: w.tables[t].rows.detach().cpu().numpy().copy() for t in check_tables}
    state0 = None if state is None else state.cpu().numpy().copy()
    say(f"[bwd] {label}: {w.num_indices} lookups, {optimizer}; backward on the GPU")
    with eb.eb_create_tables(w.tables) as h:
        eb.eb_backward_update(h, w.indices, w.offsets, w.weights, w.pooling, grad, optimizer, lr, eps, state)
        torch.cuda.synchronize()
    after = {t: w.tables[t].rows.detach().cpu().numpy() for t in check_tables}
    state1 = None if state is None else state.cpu().numpy()
    say(f"[bwd] {label}: oracle on tables {check_tables}")
    tabs = [OracleTable(before[t] if t in before else None, tb.dim, tb.dtype, tb.num_rows)
            for t, tb in enumerate(w.tables)]
    st_or = None if state0 is None else state0.copy()
    rep = ebo_backward_update(tabs, w.indices.cpu().numpy(), w.offsets.cpu().numpy(),
                              None if w.weights is None else w.weights.cpu().numpy(), w.pooling,
                              grad.cpu().numpy(), optimizer, lr, eps, st_or, report=check_tables)
    base = np.concatenate([[0], np.cumsum(R)])
    for t in check_tables:
        tb = w.tables[t]
        rows, G, S, n = rep[t]
        ref = tabs[t].rows  # updated in place by the oracle
        got = after[t]
        untouched = np.ones(tb.num_rows, bool)
        untouched[rows] = False
        raw = np.uint16 if tb.dtype == "f16" else np.uint32
        assert np.array_equal(got[untouched].view(raw), before[t][untouched].view(raw)), f"{label} t{t}: untouched rows"
        if optimizer != "sgd":
            assert np.array_equal(state1[base[t]:base[t + 1]][untouched], state0[base[t]:base[t + 1]][untouched])
        if rows.size == 0:
            continue
        _check_rows(f"{label} t{t}", tb.dtype, tb.dim, got[rows], ref[rows], G, S, n, optimizer, lr, eps,
                    None if st_or is None else st_or[base[t] + rows],
                    None if state1 is None else state1[base[t] + rows])


def _check_rows(label, dtype, D, got, ref, G, S, n, optimizer, lr, eps, s_new, s_got):
    """The bounds of the module docstring for the touched rows of one table:
    got/ref their values after the GPU's and the oracle's step, G, S, n the
    oracle's gradient, error scale and count, s_new/s_got the oracle's and the
    GPU's new Adagrad state."""
    g64 = got.astype(np.float64)
    r64 = ref.astype(np.float64)
    dG = (n[:, None] + 8) * U * S
    store = (2 * U * np.abs(r64)) if dtype == "f32" else _ulp16(r64)
    if optimizer == "sgd":
        bound = lr * dG + store
    else:
        s_new = s_new.astype(np.float64)
        ds = 2 * (np.abs(G) * dG).sum(axis=1) / D + (D + 8) * U * s_new
        scale = lr / (np.sqrt(s_new) + eps)
        # relative error of the step size lr / (sqrt(s) + eps) when the
        # state is off by at most ds (valid for any ds; module docstring),
        # plus its own roundings
        sq, sq_lo = np.sqrt(s_new), np.sqrt(np.maximum(s_new - ds, 0.0))
        with np.errstate(divide="ignore", invalid="ignore"):
            rel = np.where(s_new > 0, ds / (sq + sq_lo) / (sq_lo + eps), 0.0)
        rel = rel + 6 * U / (1 - 6 * U) * (1 + rel)
        moved = np.any(G != 0, axis=1)  # a zero gradient moves nothing, whatever the step size
        bound = scale[:, None] * dG + np.where(moved[:, None], np.abs(scale[:, None] * G) * rel[:, None], 0.0) \
            + store
        np.testing.assert_array_less(np.abs(s_got - s_new), ds + 2 * U * s_new + 1e-30)
    err = np.abs(g64 - r64)
    bound = bound / (1 - (n[:, None] + 16) * U)  # first order -> rigorous (module docstring)
    bad = err > bound + 1e-30
    assert not bad.any(), (f"{label}: {bad.sum()} elements beyond the bound; worst ratio "
                           f"{np.max(err / np.maximum(bound, 1e-30)):.3g}")


def run_and_check_touched(w, dev, optimizer, lr=0.05, eps=1e-4, label="", samples=200000):
    """run_and_check for tables too large to copy whole: the oracle steps
    compact tables holding only the rows the batch touches (the indices
    renumbered to match; a row's update depends on its own occurrences only),
    and the GPU's untouched rows are checked on a random sample."""
    T = w.num_tables
    grad = _grad(w, dev)
    R = [t.num_rows for t in w.tables]
    base = np.concatenate([[0], np.cumsum(R)])
    off = w.offsets.cpu().numpy()
    idx = w.indices.cpu().numpy()
    touched, compact_idx, sample = [], np.empty_like(idx), []
    rng = np.random.default_rng(3)
    for t in range(T):
        lo, hi = int(off[t * w.batch]), int(off[(t + 1) * w.batch])
        rows = np.unique(idx[lo:hi])
        touched.append(rows)
        compact_idx[lo:hi] = np.searchsorted(rows, idx[lo:hi])
        cand = rng.integers(0, R[t], min(samples, R[t]))
        sample.append(np.setdiff1d(cand, rows))
    state = None
    if optimizer == "rowwise_adagrad":
        gs = torch.Generator(device=dev)
        gs.manual_seed(11)
        state = torch.rand(sum(R), generator=gs, device=dev, dtype=torch.float32)

    def take(t, rows):
        return w.tables[t].rows.index_select(0, torch.from_numpy(rows).to(dev)).cpu().numpy()

    def take_state(t, rows):
        return state.index_select(0, torch.from_numpy(rows + base[t]).to(dev)).cpu().numpy()

    before = [take(t, touched[t]) for t in range(T)]
    before_s = [take(t, sample[t]) for t in range(T)]
    st0 = None if state is None else [take_state(t, touched[t]) for t in range(T)]
    st0_s = None if state is None else [take_state(t, sample[t]) for t in range(T)]
    say(f"[bwd] {label}: {w.num_indices} lookups into {R} rows, {optimizer}; backward on the GPU")
    with eb.eb_create_tables(w.tables) as h:
        eb.eb_backward_update(h, w.indices, w.offsets, w.weights, w.pooling, grad, optimizer, lr, eps, state)
        torch.cuda.synchronize()
    say(f"[bwd] {label}: oracle on the touched rows")
    tabs = [OracleTable(before[t].copy(), tb.dim, tb.dtype, len(touched[t])) for t, tb in enumerate(w.tables)]
    st_or = None if state is None else np.concatenate(st0).astype(np.float32)
    rep = ebo_backward_update(tabs, compact_idx, off, None if w.weights is None else w.weights.cpu().numpy(),
                              w.pooling, grad.cpu().numpy(), optimizer, lr, eps, st_or, report=list(range(T)))
    cbase = np.concatenate([[0], np.cumsum([len(r) for r in touched])])
    for t, tb in enumerate(w.tables):
        raw = np.uint16 if tb.dtype == "f16" else np.uint32
        assert np.array_equal(take(t, sample[t]).view(raw), before_s[t].view(raw)), f"{label} t{t}: untouched rows"
        if state is not None:
            assert np.array_equal(take_state(t, sample[t]), st0_s[t]), f"{label} t{t}: untouched state"
        rows, G, S, n = rep[t]
        assert np.all(np.diff(rows) > 0) and (rows.size == 0 or rows[-1] < len(touched[t]))
        if rows.size == 0:
            continue
        got = take(t, touched[t][rows])
        _check_rows(f"{label} t{t}", tb.dtype, tb.dim, got, tabs[t].rows[rows], G, S, n, optimizer, lr, eps,
                    None if st_or is None else st_or[cbase[t] + rows],
                    None if state is None else take_state(t, touched[t][rows]))


REDUCED = {
    "c1": {},
    "c2": dict(rows_cap=20000, batch=256),
    "c3a": dict(rows_cap=50000, batch=256),
    "c3b": dict(rows_cap=50000, batch=256),
    "c4": dict(rows_cap=20000, batch=96),
}


@pytest.mark.parametrize("optimizer", ["sgd", "rowwise_adagrad"])
@pytest.mark.parametrize("name", list(REDUCED))
def test_reduced_configs(dev, name, optimizer):
    w = make_workload(name, dev, **REDUCED[name])
    run_and_check(w, dev, optimizer, label=f"reduced {name}")


@pytest.mark.parametrize("chunks", ["2", "3", "4", "16"])
@pytest.mark.parametrize("name", ["c2", "c3b", "c4"])
def test_multi_chunk_tiles(dev, monkeypatch, name, chunks):
    # tiles of several 64-position chunks: runs that end exactly at a chunk
    # boundary inside a tile, and runs that cross chunks
    monkeypatch.setenv("EB_BWD_TILE_CHUNKS", chunks)
    w = make_workload(name, dev, **REDUCED[name])
    run_and_check(w, dev, "rowwise_adagrad", label=f"{chunks} chunks {name}")


@pytest.mark.parametrize("name", ["c2", "c4"])
def test_int32_indices(dev, name):
    w = make_workload(name, dev, index_dtype=torch.int32, **REDUCED[name])
    run_and_check(w, dev, "rowwise_adagrad", label=f"int32 {name}")


@pytest.mark.parametrize("chunks", ["1", "3"])
def test_hot_row_spans_many_tiles(dev, monkeypatch, chunks):
    monkeypatch.setenv("EB_BWD_TILE_CHUNKS", chunks)
    # one row read 5000 times (about 80 tiles of 64 positions), next to short runs
    g = torch.Generator(device="cpu")
    g.manual_seed(1)
    B = 64
    lens = torch.full((B,), 100, dtype=torch.int64)
    idx = torch.randint(0, 300, (B * 100,), generator=g)
    idx[torch.rand(B * 100, generator=g) < 0.8] = 17
    off = torch.zeros(B + 1, dtype=torch.int64)
    torch.cumsum(lens, 0, out=off[1:])
    rows = torch.randn((300, 64), generator=g).to(dev)
    w = Workload("hot", [Table(rows, 64, "f32")], B, idx.to(dev), off.to(dev), None, "sum", lens.to(dev))
    run_and_check(w, dev, "rowwise_adagrad", label="hot row")
    w.tables[0].rows.copy_(torch.randn((300, 64), generator=g).to(dev))
    run_and_check(w, dev, "sgd", label="hot row sgd")


def test_hot_rows_of_every_lane_grouping(dev, monkeypatch):
    # The fix-up adds a crossing run's tile partials with 64/L lane groups
    # (L lanes hold a row's columns 4 at a time): fp16 D32 (8 groups), fp16
    # D128 (2), fp32 D256 (1) and fp32 D64 (4), each with one row hot enough
    # to span far more than 64 tiles of 64 positions; the fp32 D64 table's
    # row spans more than 4160 tiles, past the first coarse step of the
    # search for the run's last tile.
    monkeypatch.setenv("EB_BWD_TILE_CHUNKS", "1")
    g = torch.Generator(device="cpu")
    g.manual_seed(4)
    B = 3000
    specs = [("f16", 32, 400, 12), ("f16", 128, 400, 12), ("f32", 256, 400, 12), ("f32", 64, 500, 100)]
    tables, lens_all, idx_all = [], [], []
    for dtype, D, R, L in specs:
        rows = torch.randn((R, D), generator=g)
        tables.append(Table((rows * 0.1).half().to(dev) if dtype == "f16" else rows.to(dev), D, dtype))
        lens = torch.randint(0, 2 * L + 1, (B,), generator=g)
        n = int(lens.sum())
        idx = torch.randint(0, R, (n,), generator=g)
        idx[torch.rand(n, generator=g) < 0.95] = R // 3
        lens_all.append(lens)
        idx_all.append(idx)
    lens = torch.cat(lens_all)
    off = torch.zeros(lens.numel() + 1, dtype=torch.int64)
    torch.cumsum(lens, 0, out=off[1:])
    hot = int((idx_all[-1] == specs[-1][2] // 3).sum())
    assert hot > 64 * 4160, hot
    w = Workload("hot rows", tables, B, torch.cat(idx_all).to(dev), off.to(dev), None, "mean", lens.to(dev))
    run_and_check(w, dev, "rowwise_adagrad", label="hot rows of every lane grouping")


def test_mixed_storage_and_widths(dev):
    g = torch.Generator(device="cpu")
    g.manual_seed(2)
    tables = [Table(torch.randn((500, 4), generator=g).to(dev), 4, "f32"),
              Table((torch.randn((400, 256), generator=g) * 0.01).half().to(dev), 256, "f16"),
              Table(torch.randn((300, 40), generator=g).to(dev), 40, "f32"),
              Table((torch.randn((200, 8), generator=g) * 0.01).half().to(dev), 8, "f16")]
    B = 50
    lens = torch.randint(0, 150, (4 * B,), generator=g)
    lens[:5] = 0
    off = torch.zeros(4 * B + 1, dtype=torch.int64)
    torch.cumsum(lens, 0, out=off[1:])
    parts = [torch.randint(0, t.num_rows, (int(lens[i * B:(i + 1) * B].sum()),), generator=g)
             for i, t in enumerate(tables)]
    idx = torch.cat(parts)
    wts = torch.rand(idx.numel(), generator=g)
    for pooling, weights in (("sum", wts), ("mean", None)):
        w = Workload("mixed", tables, B, idx.to(dev), off.to(dev), None if weights is None else weights.to(dev),
                     pooling, lens.to(dev))
        run_and_check(w, dev, "rowwise_adagrad", label=f"mixed {pooling}")


def test_many_tables(dev):
    # 700 tables: the scan that finds each table's first tile runs on one
    # workgroup with several tables per thread; whole tables without a
    # lookup, and empty bags, sit between tables with lookups
    g = torch.Generator(device="cpu")
    g.manual_seed(5)
    T, B = 700, 6
    tables = []
    for t in range(T):
        R = int(torch.randint(20, 200, (1,), generator=g))
        D = [4, 8, 16, 64][t % 4]
        if t % 3 == 1:  # fp16 rows take dims that are multiples of 8
            D = max(D, 8)
            tables.append(Table((torch.randn((R, D), generator=g) * 0.01).half().to(dev), D, "f16"))
        else:
            tables.append(Table(torch.randn((R, D), generator=g).to(dev), D, "f32"))
    lens = torch.randint(0, 30, (T * B,), generator=g)
    for t in range(0, T, 7):
        lens[t * B:(t + 1) * B] = 0
    off = torch.zeros(T * B + 1, dtype=torch.int64)
    torch.cumsum(lens, 0, out=off[1:])
    parts = [torch.randint(0, t.num_rows, (int(lens[i * B:(i + 1) * B].sum()),), generator=g)
             for i, t in enumerate(tables)]
    idx = torch.cat(parts)
    w = Workload("many tables", tables, B, idx.to(dev), off.to(dev), None, "sum", lens.to(dev))
    run_and_check(w, dev, "rowwise_adagrad", label="700 tables")


def test_deterministic(dev):
    w = make_workload("c3b", dev, **REDUCED["c3b"])
    init = [t.rows.clone() for t in w.tables]
    grad = _grad(w, dev)
    res = []
    for _ in range(2):
        for t, r in zip(w.tables, init):
            t.rows.copy_(r)
        st = torch.zeros(sum(t.num_rows for t in w.tables), device=dev)
        with eb.eb_create_tables(w.tables) as h:
            eb.eb_backward_update(h, w.indices, w.offsets, w.weights, w.pooling, grad, "rowwise_adagrad", 0.1, 1e-3,
                                  st)
            torch.cuda.synchronize()
        res.append(([t.rows.clone() for t in w.tables], st.clone()))
    for a, b in zip(res[0][0], res[1][0]):
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    assert torch.equal(res[0][1], res[1][1])


@pytest.mark.parametrize("name", ["c3a", "c4"])
def test_full_size(dev, name):
    say(f"[bwd] full {name}: generating")
    w = make_workload(name, dev)
    T = w.num_tables
    run_and_check(w, dev, "rowwise_adagrad", check_tables=sorted({0, T // 2, T - 1}), label=f"full {name}")


def test_checked_mode_reports_bad_data(dev, monkeypatch):
    # An index outside its table gets the table's sentinel key and updates
    # nothing; offsets that are not a partition are clamped.  Checked mode
    # reports both, and a valid call afterwards reports nothing (the error word
    # is cleared).  The broken offsets here still cover every position.
    monkeypatch.setenv("EB_CHECK", "1")
    g = torch.Generator(device="cpu")
    g.manual_seed(9)
    rows = torch.randn((10, 16), generator=g).to(dev)
    grad = torch.randn((3, 16), generator=g).to(dev)
    ok_idx = torch.tensor([1, 2, 3, 4], device=dev)
    off = torch.tensor([0, 2, 2, 4], device=dev)
    with eb.eb_create_tables([Table(rows, 16, "f32")]) as h:
        eb.eb_backward_update(h, ok_idx, off, None, "sum", grad, "sgd", 0.1)
        for bad_idx in ([1, 10, 3, 4], [1, -1, 3, 4]):
            with pytest.raises(eb.EBError) as e:
                eb.eb_backward_update(h, torch.tensor(bad_idx, device=dev), off, None, "sum", grad, "sgd", 0.1)
            assert e.value.status == eb.EB_ERR_INDEX_OOB
        for bad_off in ([0, 3, 2, 4], [0, 2, 2, 9]):
            with pytest.raises(eb.EBError) as e:
                eb.eb_backward_update(h, ok_idx, torch.tensor(bad_off, device=dev), None, "sum", grad, "sgd", 0.1)
            assert e.value.status == eb.EB_ERR_OFFSETS
        before = rows.cpu().numpy().copy()
        eb.eb_backward_update(h, ok_idx, off, None, "sum", grad, "sgd", 0.1)  # no error left over
        torch.cuda.synchronize()
    # that last step, against the oracle
    tabs = [OracleTable(before, 16, "f32", 10)]
    ebo_backward_update(tabs, np.array([1, 2, 3, 4]), np.array([0, 2, 2, 4]), None, "sum", grad.cpu().numpy(), "sgd",
                        0.1, 0.0, None, report=[0])
    got = rows.cpu().numpy()
    np.testing.assert_allclose(got, tabs[0].rows, rtol=0, atol=1e-6)
    untouched = [0, 5, 6, 7, 8, 9]  # rows no index reads keep their bits
    assert np.array_equal(got[untouched].view(np.uint32), before[untouched].view(np.uint32))


def test_backward_argument_errors(dev):
    g = torch.Generator(device="cpu")
    g.manual_seed(3)
    t8 = torch.randint(0, 255, (10, 20), generator=g, dtype=torch.uint8).to(dev)
    idx = torch.tensor([1, 2], device=dev)
    off = torch.tensor([0, 1, 2], device=dev)
    with eb.eb_create_tables([Table(t8, 16, "int8_rowwise")]) as h:
        with pytest.raises(eb.EBError) as e:
            eb.eb_backward_update(h, idx, off, None, "sum", torch.zeros((2, 16), device=dev))
        assert e.value.status == eb.EB_ERR_UNSUPPORTED
    wide = torch.zeros((10, 512), device=dev)
    with eb.eb_create_tables([Table(wide, 512, "f32")]) as h:
        with pytest.raises(eb.EBError) as e:
            eb.eb_backward_update(h, idx, off, None, "sum", torch.zeros((2, 512), device=dev))
        assert e.value.status == eb.EB_ERR_UNSUPPORTED
    tab = torch.zeros((10, 16), device=dev)
    with eb.eb_create_tables([Table(tab, 16, "f32")]) as h:
        gr = torch.zeros((2, 16), device=dev)
        with pytest.raises(eb.EBError) as e:  # Adagrad without state
            eb.eb_backward_update(h, idx, off, None, "sum", gr, "rowwise_adagrad")
        assert e.value.status == eb.EB_ERR_INVALID_ARG
        with pytest.raises(eb.EBError) as e:  # state of the wrong length
            eb.eb_backward_update(h, idx, off, None, "sum", gr, "rowwise_adagrad", optimizer_state=torch.zeros(9, device=dev))
        assert e.value.status == eb.EB_ERR_SHAPE
        with pytest.raises(eb.EBError) as e:
            eb.eb_backward_update(h, idx, off, None, "sum", torch.zeros((3, 16), device=dev))
        assert e.value.status == eb.EB_ERR_SHAPE
        with pytest.raises(eb.EBError) as e:  # workspace too small
            eb.eb_backward_update(h, idx, off, None, "sum", gr, workspace=torch.empty(16, dtype=torch.uint8, device=dev))
        assert e.value.status == eb.EB_ERR_INVALID_ARG
        need = eb.eb_backward_workspace_size(h, idx.numel())
        with pytest.raises(eb.EBError) as e:  # a float workspace counts its bytes: one float short
            eb.eb_backward_update(h, idx, off, None, "sum", gr,
                                  workspace=torch.empty((need + 3) // 4 - 1, dtype=torch.float32, device=dev))
        assert e.value.status == eb.EB_ERR_INVALID_ARG
        with pytest.raises(ValueError):
            eb.eb_backward_update(h, idx, off, None, "sum", gr,
                                  workspace=torch.empty((need + 8) * 2, dtype=torch.uint8, device=dev)[::2])
        torch.cuda.synchronize()
        assert torch.all(tab == 0)
        # a float workspace of enough bytes is accepted, and the step runs
        eb.eb_backward_update(h, idx, off, None, "sum", torch.ones((2, 16), device=dev), learning_rate=0.5,
                              workspace=torch.empty((need + 3) // 4, dtype=torch.float32, device=dev))
        torch.cuda.synchronize()
        assert torch.all(tab[1:3] == -0.5) and torch.all(tab[0] == 0) and torch.all(tab[3:] == 0)


def _sort_shape_workload(dev, row_counts, B, weighted, seed):
    """fp32 D4 tables of the given row counts.  Each table's bags (lengths
    U{0..300}) draw half their indices from 8 hot rows spread over the whole
    range and half uniformly, so runs are long and short and every digit of
    every sort pass varies."""
    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    gd = torch.Generator(device=dev)
    gd.manual_seed(seed)
    tables, lens_all, idx_all = [], [], []
    for R in row_counts:
        tables.append(Table(torch.randn((R, 4), generator=gd, device=dev), 4, "f32"))
        lens = torch.randint(0, 301, (B,), generator=g)
        n = int(lens.sum())
        hot = torch.randint(0, R, (8,), generator=g)
        idx = torch.randint(0, R, (n,), generator=g)
        pick = torch.rand(n, generator=g) < 0.5
        idx[pick] = hot[torch.randint(0, 8, (int(pick.sum()),), generator=g)]
        lens_all.append(lens)
        idx_all.append(idx)
    lens = torch.cat(lens_all)
    off = torch.zeros(lens.numel() + 1, dtype=torch.int64)
    torch.cumsum(lens, 0, out=off[1:])
    idx = torch.cat(idx_all)
    wts = torch.rand(idx.numel(), generator=g).to(dev) if weighted else None
    return Workload("sort shape", tables, B, idx.to(dev), off.to(dev), wts, "sum", lens.to(dev))


# (row counts, weighted): the sort's digits cover the rows of the largest
# table (its row count included, the sentinel), in passes of up to 9 bits;
# unweighted elements hold the row and the table-local bag id in 32 bits when
# both fit, weighted ones the row and the position.
SORT_SHAPES = {
    "1 pass (9 bits)": ([300, 511], False),
    "2 passes of 9 bits": ([512, 70000], False),
    "3 passes of 9 bits, 32-bit elements": ([20_000_000, 1000], False),
    "3 passes of 9 bits, 64-bit elements": ([20_000_000, 1000], True),
    "4 passes of 7 bits": ([150_000_000, 3], False),
}


@pytest.mark.parametrize("shape", list(SORT_SHAPES))
def test_sort_digit_shapes(dev, shape):
    counts, weighted = SORT_SHAPES[shape]
    w = _sort_shape_workload(dev, counts, 64, weighted, seed=len(shape))
    run_and_check_touched(w, dev, "rowwise_adagrad", label=shape)


@pytest.mark.parametrize("items", ["4", "8", "12", "16"])
def test_sort_block_sizes(dev, monkeypatch, items):
    # every elements-per-thread choice of the sort on a 3-pass sort whose
    # tables span several blocks of each size
    monkeypatch.setenv("EB_BWD_SORT_ITEMS", items)
    w = _sort_shape_workload(dev, [20_000_000, 70000, 1000], 256, False, seed=9)
    run_and_check_touched(w, dev, "rowwise_adagrad", label=f"{items} items per thread")
