"""GPU parity of the un-pooled (sequence) lookup, eb_forward_seq, against the
oracle through the C ABI.

Every output element is one exact conversion of a table element (one
rounding for int8 row-wise rows), so the bar is bit equality, element by
element, at reduced sizes and on sampled positions at full size.
"""
import numpy as np
import pytest
import torch

from conftest import compact_oracle_table, oracle_tables
from oracle import OracleTable, ebo_forward_seq
from paper_2609_30656_amd import eb
from paper_2609_30656_amd.workload import make_workload
from test_parity_gpu import REDUCED, WIDTHS, _custom, _table

pytestmark = pytest.mark.gpu


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


def seq_numel(w):
    off = w.offsets.cpu().numpy()
    B = w.batch
    return sum(int(off[(t + 1) * B] - off[t * B]) * tb.dim for t, tb in enumerate(w.tables))


def run_seq(w, numel=None):
    n = seq_numel(w) if numel is None else numel
    out = torch.full((n,), float("nan"), dtype=torch.float32, device=w.indices.device)
    with eb.eb_create_tables(w.tables) as h:
        eb.eb_forward_seq(h, w.indices, w.offsets, out)
        torch.cuda.synchronize()
    return out


def full_seq_check(w, label):
    got = run_seq(w).cpu().numpy()
    ref = ebo_forward_seq(oracle_tables(w), w.indices.cpu().numpy(), w.offsets.cpu().numpy())
    assert got.shape == ref.shape
    same = got.view(np.uint32) == ref.view(np.uint32)
    assert same.all(), f"{label}: {np.count_nonzero(~same)} of {same.size} elements differ"


@pytest.mark.parametrize("name", list(REDUCED))
def test_reduced_configs(dev, name):
    say(f"[seq] reduced {name}")
    full_seq_check(make_workload(name, dev, **REDUCED[name]), f"reduced {name}")


@pytest.mark.parametrize("variant", ["int64", "int32"])
def test_c5_split_int8_layout(dev, variant):
    say(f"[seq] c5 split layout {variant}")
    kw = dict(REDUCED["c5"], int8_layout="split")
    if variant == "int32":
        kw["index_dtype"] = torch.int32
    full_seq_check(make_workload("c5", dev, **kw), f"c5 split {variant}")


@pytest.mark.parametrize("name", ["c2", "c4", "c5"])
def test_int32_indices(dev, name):
    say(f"[seq] int32 {name}")
    full_seq_check(make_workload(name, dev, index_dtype=torch.int32, **REDUCED[name]), f"int32 {name}")


@pytest.mark.parametrize("k", ["1", "2", "5", "32"])
@pytest.mark.parametrize("name", ["c3b", "c4"])
def test_chunks_per_wave(dev, monkeypatch, name, k):
    # spans of several chunks that start and end inside tables and cross
    # table boundaries (c4: 100 tables of four widths)
    say(f"[seq] chunks per wave {k} {name}")
    monkeypatch.setenv("EB_BAGS_PER_WAVE", k)
    full_seq_check(make_workload(name, dev, **REDUCED[name]), f"k={k} {name}")


@pytest.mark.parametrize("k", ["1", "3"])
def test_every_width_and_empty_tables(dev, monkeypatch, k):
    say(f"[seq] widths k={k}")
    monkeypatch.setenv("EB_BAGS_PER_WAVE", k)
    rng = np.random.default_rng(9)
    tables = [_table(dev, dt, 300 + 7 * i, D, seed=i) for i, (dt, D) in enumerate(WIDTHS)]
    B = 11
    lens = [rng.integers(0, 20, B) for _ in tables]
    lens[3][:] = 0  # an empty table
    lens[4][:] = 0
    lens[5][:] = [0] * (B - 1) + [1]  # one position
    w = _custom(dev, tables, lens)
    full_seq_check(w, f"widths k={k}")


def test_padded_row_strides(dev):
    say("[seq] padded strides")
    tables = [_table(dev, "f32", 500, 64, stride=512), _table(dev, "f16", 500, 64, stride=256),
              _table(dev, "int8_rowwise", 500, 128, stride=144), _table(dev, "int8_rowwise", 500, 32, stride=40),
              _table(dev, "int8_rowwise_split", 500, 128, stride=160, seed=1),
              _table(dev, "int8_rowwise_split", 500, 32, stride=48, seed=2)]
    rng = np.random.default_rng(6)
    full_seq_check(_custom(dev, tables, [rng.integers(0, 50, 64) for _ in tables]), "padded strides")


def test_no_indices(dev):
    say("[seq] N = 0")
    tables = [_table(dev, "f16", 50, 64, seed=t) for t in range(3)]
    w = _custom(dev, tables, [np.zeros(5, np.int64) for _ in tables])
    out = torch.empty(0, device=dev)
    with eb.eb_create_tables(w.tables) as h:
        eb.eb_forward_seq(h, w.indices, w.offsets, out)


@pytest.mark.parametrize("name", ["c2", "c3a", "c4"])
def test_full_size_every_element(dev, name):
    say(f"[seq] full {name}")
    full_seq_check(make_workload(name, dev), f"full {name}")


@pytest.mark.parametrize("layout", ["packed", "split"])
def test_full_c5_sampled(dev, layout):
    say(f"[seq] full c5 ({layout} int8 rows): generating")
    w = make_workload("c5", dev, int8_layout=layout)
    n = w.num_indices
    say(f"[seq] full c5: {n} positions, {n * 128 * 4 / 1e9:.1f} GB of output")
    out = run_seq(w).view(n, 128)
    assert not torch.isnan(out[::9973]).any()
    rng = np.random.default_rng(2)
    pos = np.unique(np.concatenate([[0, n - 1], rng.choice(n, 3000, replace=False)]))
    B = w.batch
    starts = w.offsets[::B].cpu().numpy()  # table starts, [T + 1]
    tabs = np.searchsorted(starts, pos, side="right") - 1
    got = out[torch.from_numpy(pos).to(dev)].cpu().numpy()
    idx = w.indices[torch.from_numpy(pos).to(dev)].cpu().numpy()
    for t in np.unique(tabs):
        sel = np.nonzero(tabs == t)[0]
        rows, inv = np.unique(idx[sel], return_inverse=True)
        ref = ebo_forward_seq([compact_oracle_table(w.tables[t], rows)],
                              inv.astype(np.int64), np.array([0, inv.size], np.int64)).reshape(-1, 128)
        assert np.array_equal(got[sel].view(np.uint32), ref.view(np.uint32)), f"table {t}"


def test_argument_errors(dev):
    say("[seq] argument errors")
    w = make_workload("c2", dev, rows_cap=1000, batch=8, num_tables=3)
    n, D = w.num_indices, 64
    with eb.eb_create_tables(w.tables) as h:
        for out, status in [(torch.empty(n * D + 4, device=dev), eb.EB_ERR_SHAPE),
                            (torch.empty(n * D, device=dev, dtype=torch.int32), eb.EB_ERR_DTYPE),
                            (torch.empty(n * D + 1, device=dev)[1:], eb.EB_ERR_UNSUPPORTED)]:
            with pytest.raises(eb.EBError) as e:
                eb.eb_forward_seq(h, w.indices, w.offsets, out)
            assert e.value.status == status
        with pytest.raises(eb.EBError) as e:
            eb.eb_forward_seq(h, w.indices, w.offsets[:-1], torch.empty(n * D, device=dev))
        assert e.value.status == eb.EB_ERR_SHAPE
    mixed = [_table(dev, "f32", 10, 8), _table(dev, "f32", 10, 16)]
    wk = _custom(dev, mixed, [np.full(3, 2, np.int64) for _ in mixed])
    with eb.eb_create_tables(wk.tables) as h:
        with pytest.raises(eb.EBError) as e:  # outside [N * 8, N * 16]
            eb.eb_forward_seq(h, wk.indices, wk.offsets, torch.empty(12 * 16 + 4, device=dev))
        assert e.value.status == eb.EB_ERR_SHAPE


def test_checked_mode(dev, monkeypatch):
    say("[seq] checked mode")
    monkeypatch.setenv("EB_CHECK", "1")
    mixed = [_table(dev, "f32", 10, 8, seed=0), _table(dev, "f32", 10, 16, seed=1)]
    wk = _custom(dev, mixed, [np.full(3, 2, np.int64) for _ in mixed])  # N = 12, exact size 6*8 + 6*16
    with eb.eb_create_tables(wk.tables) as h:
        out = torch.empty(6 * 8 + 6 * 16, device=dev)
        eb.eb_forward_seq(h, wk.indices, wk.offsets, out)
        with pytest.raises(eb.EBError) as e:  # within the host's range, but too small for these offsets
            eb.eb_forward_seq(h, wk.indices, wk.offsets, torch.empty(6 * 8 + 6 * 16 - 16, device=dev))
        assert e.value.status == eb.EB_ERR_SHAPE
        bad = wk.indices.clone()
        bad[7] = 10  # one past the end of table 1
        with pytest.raises(eb.EBError) as e:
            eb.eb_forward_seq(h, bad, wk.offsets, out)
        assert e.value.status == eb.EB_ERR_INDEX_OOB
