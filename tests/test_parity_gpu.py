"""GPU parity: libeb's HIP path against the CPU oracle, through the C ABI.

Bar (per output element of a bag with L lookups, oracle value o, GPU value g,
and the oracle's error scale s = sum_i |w_i x_i| (divided by L for mean)):
  * L <= 1: g and o have the same bits (a gather, or an empty bag = +0.0);
  * otherwise |g - o| <= rtol * s with rtol = 1e-5 for fp32 tables and 2e-3
    for fp16 / int8 row-wise tables;
  * and, tighter, the a-priori bound of fp32 summation in any order,
    |g - o| <= (L + 3) * 2^-24 * s' + 2 * 2^-24 * s, where s' = s except for
    unweighted int8 row-wise tables: the kernel sums s*q and the biases c
    separately (a reassociation), so s' = sum_i (|s_i q_i| + |c_i|), the sum
    of the oracle's fp64 absolute sums over a table of |s| q and over a table
    of |c| (both exact in fp32).
"""
import os

import numpy as np
import pytest
import torch

from conftest import oracle_forward, oracle_tables, ulp_distance
from oracle import OracleTable, ebo_forward
from paper_2609_30656_amd import eb
from paper_2609_30656_amd.workload import Table, make_workload

pytestmark = pytest.mark.gpu

RTOL = {"f32": 1e-5, "f16": 2e-3, "int8_rowwise": 2e-3, "int8_rowwise_split": 2e-3}
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


def run_gpu(w, stream=None, prefill=float("nan")):
    out = torch.full((w.batch, w.sum_dim), prefill, dtype=torch.float32, device=w.indices.device)
    with eb.eb_create_tables(w.tables, stream) as h:
        eb.eb_forward(h, w.indices, w.offsets, w.weights, w.pooling, out)
        torch.cuda.synchronize()
    return out


def check(got, ref, asum, L, rtol, label, bscale=None):
    """got/ref fp32, asum fp64, L int (same shape); bscale: scale of the
    summation bound (asum when None)."""
    got = np.asarray(got, np.float32)
    err = np.abs(got.astype(np.float64) - ref.astype(np.float64))
    assert not np.isnan(got).any(), f"{label}: NaN in output (an element was not written)"
    short = L <= 1
    if short.any():
        same = got.view(np.uint32)[short] == ref.view(np.uint32)[short]
        assert same.all(), f"{label}: {np.count_nonzero(~same)} one-row/empty outputs not bit-exact"
    long_ = ~short
    if long_.any():
        lim = rtol * asum[long_]
        bad = err[long_] > lim
        assert not bad.any(), (f"{label}: {bad.sum()} outputs beyond rtol {rtol}; worst ratio "
                               f"{np.max(err[long_] / np.maximum(lim, 1e-300)):.3g}")
        bs = asum if bscale is None else bscale
        bound = (L[long_] + 3) * U * bs[long_] + 2 * U * asum[long_]
        over = err[long_] > bound
        assert not over.any(), f"{label}: {over.sum()} outputs beyond the summation error bound"


def per_element_lengths(w, bags=None):
    lens = w.lengths.cpu().numpy().reshape(w.num_tables, w.batch)
    if bags is None:
        return np.concatenate([np.repeat(lens[t][:, None], tb.dim, axis=1) for t, tb in enumerate(w.tables)], 1)
    return lens.reshape(-1)[bags][:, None]


def int8_parts(ot):
    """Codes [R, D] (uint8), |scale| and |bias| [R, 1] (fp32, exact) of an
    int8 row-wise OracleTable, packed (codes, then the fp16 scale and bias of
    each row) or split (codes in the rows, the scale/bias words after them)."""
    D = ot.dim
    if ot.dtype == "int8_rowwise_split":
        R, st = ot.num_rows, ot.row_stride
        buf = ot.rows.reshape(-1)
        codes, words = buf[:R * st].reshape(R, st)[:, :D], buf[R * st:R * st + 4 * R].reshape(R, 4)
    else:
        codes, words = ot.rows[:, :D], ot.rows[:, D:D + 4]
    sc = np.abs(words[:, 0:2].copy().view(np.float16).astype(np.float32))
    bi = np.abs(words[:, 2:4].copy().view(np.float16).astype(np.float32))
    return codes, sc, bi


def is_int8(dtype):
    return dtype in ("int8_rowwise", "int8_rowwise_split")


def split_scale(w, tables, bags=None):
    """Scale s' of the summation bound for unweighted int8 row-wise tables,
    whose kernel sums s*q and the biases c separately:
    s' = sum_i (|s_i q_i| + |c_i|), the oracle's fp64 absolute sums over a
    table of |s| q (exact in fp32: an 11-bit by 8-bit product) plus those over
    a table holding |c| in every column (exact).  Other tables contribute
    their own |w x| sums.  None when no table of `w` takes the split sum."""
    if w.weights is not None or not any(is_int8(t.dtype) for t in w.tables):
        return None
    prods, biases = [], []
    for tb, ot in zip(w.tables, tables):
        if ot.rows is None:
            prods.append(ot)
            biases.append(ot)
            continue
        R, D = tb.num_rows, tb.dim
        if not is_int8(tb.dtype):
            prods.append(ot)
            biases.append(OracleTable(np.zeros((R, D), np.float32), D, "f32", R))
            continue
        q, sc, bi = int8_parts(ot)
        prods.append(OracleTable(np.ascontiguousarray(q.astype(np.float32) * sc), D, "f32", R))
        biases.append(OracleTable(np.ascontiguousarray(np.broadcast_to(bi, (R, D))), D, "f32", R))
    return (oracle_forward(w, tables=prods, bags=bags)[1] + oracle_forward(w, tables=biases, bags=bags)[1])


def full_check(w, label, stream=None):
    got = run_gpu(w, stream).cpu().numpy()
    tabs = oracle_tables(w)
    ref, asum = oracle_forward(w, tables=tabs)
    bscale = split_scale(w, tabs)
    rtol = max(RTOL[t.dtype] for t in w.tables)
    check(got, ref, asum, per_element_lengths(w), rtol, label, bscale)
    return got


# ----------------------------------------------------------------------------
# every config at sizes the oracle finishes in seconds (several tiles, ragged tails)

REDUCED = {
    "c1": {},
    "c2": dict(rows_cap=20000, batch=256),
    "c3a": dict(rows_cap=50000, batch=256),
    "c3b": dict(rows_cap=50000, batch=256),
    "c4": dict(rows_cap=20000, batch=96),
    "c5": dict(rows_cap=20000, batch=128),
}


@pytest.mark.parametrize("name", list(REDUCED))
def test_reduced_configs_elementwise(dev, name):
    say(f"[parity] reduced {name} {REDUCED[name]}")
    w = make_workload(name, dev, **REDUCED[name])
    full_check(w, f"reduced {name}")


@pytest.mark.parametrize("name", ["c2", "c3b", "c4", "c5"])
def test_int32_indices(dev, name):
    say(f"[parity] int32 indices {name}")
    w = make_workload(name, dev, index_dtype=torch.int32, **REDUCED[name])
    full_check(w, f"int32 {name}")


@pytest.mark.parametrize("name", ["c2", "c5"])
def test_uniform_index_control(dev, name):
    say(f"[parity] uniform indices {name}")
    w = make_workload(name, dev, index_law="uniform", **REDUCED[name])
    full_check(w, f"uniform {name}")


@pytest.mark.parametrize("variant", ["zipf", "int32", "uniform", "k3", "k32"])
def test_c5_split_int8_layout(dev, monkeypatch, variant):
    # c5's tables in the split layout (codes in 128-byte rows, scale/bias
    # block after them): the same values as the packed layout, so the same
    # bar and the same oracle outputs
    say(f"[parity] c5 split layout, {variant}")
    kw = dict(REDUCED["c5"], int8_layout="split")
    if variant == "int32":
        kw["index_dtype"] = torch.int32
    if variant == "uniform":
        kw["index_law"] = "uniform"
    if variant.startswith("k"):
        monkeypatch.setenv("EB_BAGS_PER_WAVE", variant[1:])
    w = make_workload("c5", dev, **kw)
    assert all(t.dtype == "int8_rowwise_split" and t.row_stride_bytes == 128 for t in w.tables)
    got = full_check(w, f"c5 split {variant}")
    packed = make_workload("c5", dev, **dict(kw, int8_layout="packed"))
    assert torch.equal(packed.indices, w.indices)
    # the layout changes where the bytes are, not the values or the order of
    # the sum: the packed tables give the same bits
    assert np.array_equal(got.view(np.uint32), run_gpu(packed).cpu().numpy().view(np.uint32))


@pytest.mark.parametrize("k", [2, 3, 7, 32])
@pytest.mark.parametrize("name", ["c3a", "c4", "c5"])
def test_bags_per_wave(dev, monkeypatch, name, k):
    # several consecutive bags (and their chunk stream) per wavefront; the
    # last group of each table is partial whenever k does not divide B
    say(f"[parity] bags per wave {k} {name}")
    monkeypatch.setenv("EB_BAGS_PER_WAVE", str(k))
    monkeypatch.setenv("EB_TAIL_BAGS", "0")  # runs of k bags only (no taper)
    w = make_workload(name, dev, **REDUCED[name])
    full_check(w, f"k={k} {name}")


@pytest.mark.parametrize("remap", ["0", "1"])
@pytest.mark.parametrize("name", ["c3b", "c4"])
def test_tapered_runs(dev, monkeypatch, name, remap):
    # each table's last bags in short runs after its runs of k bags: with the
    # XCD renumbering the runs go table by table, without it every table's
    # head runs come first.  Which wavefront pools a bag changes, the order of
    # a bag's additions does not, so every mapping gives the untapered
    # output's bits (bags left to the long-bag pass are added in another
    # order: the oracle's bar then).
    say(f"[parity] tapered runs {name} remap={remap}")
    monkeypatch.setenv("EB_XCD_REMAP", remap)
    w = make_workload(name, dev, **REDUCED[name])
    monkeypatch.setenv("EB_BAGS_PER_WAVE", "3")
    monkeypatch.setenv("EB_TAIL_BAGS", "0")
    base = full_check(w, f"untapered {name}")
    ref, asum = oracle_forward(w)
    B = w.batch
    cases = [(k, tail, run, long_len)
             for k in ("3", "7") for tail in (1, 37, B - 1, B, 10 ** 9) for run in ("1", "2", "5")
             for long_len in ("0", "16")]
    for k, tail, run, long_len in cases:
        say(f"[parity]   k={k} tail={tail} run={run} long={long_len}")
        monkeypatch.setenv("EB_BAGS_PER_WAVE", k)
        monkeypatch.setenv("EB_TAIL_BAGS", str(tail))
        monkeypatch.setenv("EB_TAIL_RUN", run)
        monkeypatch.setenv("EB_LONG_BAG", long_len)
        got = run_gpu(w).cpu().numpy()
        label = f"{name} remap={remap} k={k} tail={tail} run={run} long={long_len}"
        if long_len == "0":
            assert np.array_equal(got.view(np.uint32), base.view(np.uint32)), label
        else:  # the long-bag pass adds a bag's quarters and segments: another order
            check(got, ref, asum, per_element_lengths(w), RTOL[w.tables[0].dtype], label)


@pytest.mark.parametrize("long_len,seg", [("4", "2048"), ("16", "64"), ("64", "128")])
@pytest.mark.parametrize("name", ["c1", "c2", "c3a", "c3b", "c4", "c5"])
def test_long_bag_pass(dev, monkeypatch, name, long_len, seg):
    # bags longer than EB_LONG_BAG lookups are left by the lookup kernel to
    # the long-bag pass, which pools them in segments of EB_LONG_SEG
    # positions (four wavefronts each, indices staged in LDS) and adds the
    # segments' partial rows in order; a low threshold sends most bags down
    # that path, short segments cut them into several
    say(f"[parity] long-bag pass at {long_len}, segments of {seg}, {name}")
    monkeypatch.setenv("EB_LONG_BAG", long_len)
    monkeypatch.setenv("EB_LONG_SEG", seg)
    w = make_workload(name, dev, **REDUCED[name])
    full_check(w, f"long>{long_len} seg {seg} {name}")


def test_long_bag_queue_overflow(dev, monkeypatch):
    # about 60 000 long bags of one segment each against a queue of 16 384
    # entries: the bags whose entries do not fit are pooled by the wavefront
    # that holds them, as without the pass.  Three calls on one handle, so
    # each must find the queue's counters cleared by the one before
    say("[parity] long-bag queue overflow")
    monkeypatch.setenv("EB_LONG_BAG", "4")
    monkeypatch.setenv("EB_LONG_SEG", "64")
    w = make_workload("c5", dev, rows_cap=20000, batch=1024)
    w2 = make_workload("c5", dev, rows_cap=20000, batch=96, batch_seed=1)
    lens = w.lengths.cpu().numpy()
    assert (np.ceil(lens[lens > 4] / 64)).sum() > 16384
    rtol = RTOL[w.tables[0].dtype]
    with eb.eb_create_tables(w.tables) as h:
        for rep, wl in enumerate([w, w2, w]):
            out = torch.full((wl.batch, wl.sum_dim), float("nan"), device=dev)
            eb.eb_forward(h, wl.indices, wl.offsets, wl.weights, wl.pooling, out)
            torch.cuda.synchronize()
            tabs = oracle_tables(wl)
            ref, asum = oracle_forward(wl, tables=tabs)
            check(out.cpu().numpy(), ref, asum, per_element_lengths(wl), rtol, f"overflow call {rep}",
                  split_scale(wl, tabs))


# ----------------------------------------------------------------------------
# full sizes, in the launch configuration the benchmark times

def test_full_c1(dev):
    say("[parity] full c1")
    full_check(make_workload("c1", dev), "full c1")


def test_full_c2_every_element(dev):
    say("[parity] full c2 (all 53,248 bags)")
    w = make_workload("c2", dev)
    full_check(w, "full c2")


def _sampled(w, tables_to_check, n_random=400, seed=0):
    """Bags of the given tables: random ones plus the longest, the empty and
    one-row ones, and each table's first and last bag."""
    rng = np.random.default_rng(seed)
    lens = w.lengths.cpu().numpy()
    B = w.batch
    picks = []
    for t in tables_to_check:
        g = np.arange(t * B, (t + 1) * B)
        L = lens[g]
        picks += [g[0], g[-1], g[np.argmax(L)]]
        picks += list(rng.choice(g, size=min(n_random, B), replace=False))
        for cond in (L == 0, L == 1, L >= 100):
            sel = g[cond]
            if sel.size:
                picks += list(rng.choice(sel, size=min(20, sel.size), replace=False))
    return np.unique(np.array(picks, dtype=np.int64))


@pytest.mark.parametrize("name", ["c3a", "c3b", "c4", "c5", "c5-packed"])
def test_full_size_sampled(dev, name):
    say(f"[parity] full {name}: generating")
    name, _, layout = name.partition("-")
    w = make_workload(name, dev, int8_layout=layout or None)
    T = w.num_tables
    check_tables = sorted({0, T // 2, T - 1})
    say(f"[parity] full {name}: {w.num_indices} lookups, {w.num_bags} bags; forward")
    got = run_gpu(w)
    assert not torch.isnan(got).any()
    # empty bags are +0.0 everywhere, at full size
    lens = w.lengths.view(T, w.batch)
    col = 0
    for t, tb in enumerate(w.tables):
        empty = lens[t] == 0
        if empty.any():
            z = got[empty, col:col + tb.dim]
            assert torch.equal(z.view(torch.int32), torch.zeros_like(z).view(torch.int32))
        col += tb.dim
    bags = _sampled(w, check_tables)
    say(f"[parity] full {name}: oracle on {bags.size} sampled bags of tables {check_tables}")
    tabs = [OracleTable.of(tb, with_rows=t in check_tables) for t, tb in enumerate(w.tables)]
    ref, asum = oracle_forward(w, tables=tabs, bags=bags)
    bscale = split_scale(w, tabs, bags)
    bscale = asum if bscale is None else bscale
    g_host = got.cpu().numpy()
    doff = np.concatenate([[0], np.cumsum([tb.dim for tb in w.tables])])
    B = w.batch
    L = per_element_lengths(w, bags)
    for k, g in enumerate(bags):
        t, b = divmod(int(g), B)
        D = w.tables[t].dim
        check(g_host[b, doff[t]:doff[t] + D], ref[k, :D], asum[k, :D], np.full(D, L[k, 0]),
              RTOL[w.tables[t].dtype], f"full {name} bag {g}", bscale[k, :D])


# ----------------------------------------------------------------------------
# shapes and edge cases


def _table(dev, dtype, R, D, stride=None, seed=0):
    g = torch.Generator(device=dev)
    g.manual_seed(1000 + seed)
    if dtype == "f32":
        width = D if stride is None else stride // 4
        rows = torch.rand((R, width), generator=g, device=dev) * 2 - 1
    elif dtype == "f16":
        width = D if stride is None else stride // 2
        rows = (torch.randn((R, width), generator=g, device=dev) * 0.01).half()
    elif dtype == "int8_rowwise":
        width = D + 4 if stride is None else stride
        rows = torch.randint(0, 256, (R, width), generator=g, device=dev, dtype=torch.uint8)
        sc = (torch.rand(R, generator=g, device=dev) * 3e-4 + 1e-4).half().view(torch.uint8).view(R, 2)
        bi = (torch.rand(R, generator=g, device=dev) * 0.04 - 0.06).half().view(torch.uint8).view(R, 2)
        rows[:, D:D + 2] = sc
        rows[:, D + 2:D + 4] = bi
    else:
        # the values _table draws for a packed table, stored split: codes in
        # rows of `stride` bytes (padding bytes 0xAB, never read), then the
        # rows' scale/bias words
        return to_split(_table(dev, "int8_rowwise", R, D, seed=seed), stride)
    return Table(rows, D, dtype)


def to_split(packed, stride=None):
    """A packed int8 row-wise Table's values in the split layout."""
    R, D = packed.num_rows, packed.dim
    stride = (D + 15) // 16 * 16 if stride is None else stride
    storage = torch.full((R * stride + 4 * R,), 0xAB, dtype=torch.uint8, device=packed.rows.device)
    rows = storage[:R * stride].view(R, stride)
    rows[:, :D] = packed.rows[:, :D]
    storage[R * stride:].view(R, 4).copy_(packed.rows[:, D:D + 4])
    return Table(rows, D, "int8_rowwise_split", storage)


def _custom(dev, tables, lens_per_table, weighted=False, pooling="sum", index_dtype=torch.int64, seed=0):
    from paper_2609_30656_amd.workload import Workload

    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    B = len(lens_per_table[0])
    lengths = torch.tensor(np.concatenate(lens_per_table), dtype=torch.int64)
    offsets = torch.zeros(lengths.numel() + 1, dtype=torch.int64)
    torch.cumsum(lengths, 0, out=offsets[1:])
    idx = []
    for t, tb in enumerate(tables):
        n = int(sum(lens_per_table[t]))
        idx.append(torch.randint(0, tb.num_rows, (n,), generator=g))
    indices = torch.cat(idx) if idx else torch.empty(0, dtype=torch.int64)
    weights = torch.rand(indices.numel(), generator=g) if weighted else None
    return Workload("custom", tables, B, indices.to(index_dtype).to(dev), offsets.to(index_dtype).to(dev),
                    None if weights is None else weights.to(dev), pooling, lengths.to(dev))


WIDTHS = [("f32", 4), ("f32", 12), ("f32", 20), ("f32", 100), ("f32", 260), ("f32", 1024), ("f32", 1028),
          ("f16", 8), ("f16", 24), ("f16", 40), ("f16", 136), ("f16", 520), ("f16", 2048),
          ("int8_rowwise", 16), ("int8_rowwise", 48), ("int8_rowwise", 272), ("int8_rowwise", 1024),
          ("int8_rowwise", 2064), ("int8_rowwise_split", 16), ("int8_rowwise_split", 128),
          ("int8_rowwise_split", 272), ("int8_rowwise_split", 2064)]


@pytest.mark.parametrize("k", ["0", "5"])
@pytest.mark.parametrize("mode", ["sum", "mean", "weighted"])
def test_every_width_in_one_launch(dev, monkeypatch, mode, k):
    say(f"[parity] widths {mode} k={k}")
    monkeypatch.setenv("EB_BAGS_PER_WAVE", k)
    rng = np.random.default_rng(5)
    tables = [_table(dev, dt, 300 + 7 * i, D, seed=i) for i, (dt, D) in enumerate(WIDTHS)]
    B = 37
    lens = [rng.integers(0, 140, B) for _ in tables]
    for l in lens:
        l[0], l[1], l[2] = 0, 1, 129  # empty, one row, just over two index chunks
    w = _custom(dev, tables, lens, weighted=(mode == "weighted"), pooling="mean" if mode == "mean" else "sum")
    full_check(w, f"widths {mode}")


@pytest.mark.parametrize("mode", ["sum", "mean", "weighted"])
def test_long_bag_pass_every_width(dev, monkeypatch, mode):
    # every storage type and width (1 KiB column windows included) through
    # the long-bag pass, bags of one to five segments of 64 positions
    say(f"[parity] long-bag pass, every width, {mode}")
    monkeypatch.setenv("EB_LONG_BAG", "8")
    monkeypatch.setenv("EB_LONG_SEG", "64")
    rng = np.random.default_rng(15)
    tables = [_table(dev, dt, 300 + 7 * i, D, seed=i) for i, (dt, D) in enumerate(WIDTHS)]
    lens = [rng.integers(0, 300, 13) for _ in tables]
    for l in lens:
        l[0], l[1], l[2], l[3], l[4], l[5] = 0, 1, 9, 8, 64, 65  # empty, one row, just (not) long, segment ends
    w = _custom(dev, tables, lens, weighted=(mode == "weighted"), pooling="mean" if mode == "mean" else "sum")
    full_check(w, f"long pass widths {mode}")


@pytest.mark.parametrize("long_len", ["0", "default", "4096"])
def test_one_very_long_bag(dev, monkeypatch, long_len):
    # a bag of 300 000 lookups among short ones: one wavefront per bag
    # (EB_LONG_BAG=0), or the long-bag pass for bags of more than 1024 (the
    # default here: 42 000 lookups per bag on average) or 4096 lookups, in
    # segments of 2048 positions
    say(f"[parity] one very long bag, EB_LONG_BAG={long_len}")
    if long_len == "default":
        monkeypatch.delenv("EB_LONG_BAG", raising=False)
    else:
        monkeypatch.setenv("EB_LONG_BAG", long_len)
    tables = [_table(dev, "f32", 100000, 64), _table(dev, "f16", 50000, 128, seed=1)]
    lens = [np.array([3, 300000, 0, 7, 4097, 1]), np.array([4096, 2, 200000, 0, 5, 9])]
    w = _custom(dev, tables, lens)
    got = full_check(w, "very long bag")
    if long_len == "default":  # the pass ran, at the default threshold
        monkeypatch.setenv("EB_LONG_BAG", "1024")
        assert np.array_equal(got.view(np.uint32), run_gpu(w).cpu().numpy().view(np.uint32))


def test_long_bag_pass_by_default(dev, monkeypatch):
    # without EB_LONG_BAG the pass runs for batches of at least 2^23 lookups
    # (or of 64 lookups per bag on average): a batch of 8.4 M lookups with
    # bags of 1 000 000, 4097 and 1025 lookups among bags of about twenty
    # gives the bits of EB_LONG_BAG=1024 and matches the oracle; a batch of
    # 400 000 lookups in bags of about twenty, one of 5000, gives the bits of
    # EB_LONG_BAG=0 (no pass)
    say("[parity] long-bag pass by default")
    rng = np.random.default_rng(21)
    table = _table(dev, "f32", 100000, 16)
    for B, long_lens, same_as in [(380000, [1_000_000, 4097, 1025, 1024], "1024"), (20000, [5000], "0")]:
        monkeypatch.delenv("EB_LONG_BAG", raising=False)
        lens = rng.integers(10, 31, B)
        lens[:len(long_lens)] = long_lens
        rng.shuffle(lens)
        big = lens.sum() >= 1 << 23
        assert big == (same_as == "1024") and lens.mean() < 64
        w = _custom(dev, [table], [lens])
        got = full_check(w, f"default, B={B}")
        monkeypatch.setenv("EB_LONG_BAG", same_as)
        assert np.array_equal(got.view(np.uint32), run_gpu(w).cpu().numpy().view(np.uint32)), B


def test_padded_row_strides(dev):
    say("[parity] padded strides")
    tables = [_table(dev, "f32", 500, 64, stride=512), _table(dev, "f16", 500, 64, stride=256),
              _table(dev, "int8_rowwise", 500, 128, stride=144), _table(dev, "int8_rowwise", 500, 32, stride=40),
              _table(dev, "int8_rowwise_split", 500, 128, stride=160, seed=1),
              _table(dev, "int8_rowwise_split", 500, 32, stride=48, seed=2)]
    rng = np.random.default_rng(6)
    w = _custom(dev, tables, [rng.integers(0, 50, 64) for _ in tables], weighted=True)
    full_check(w, "padded strides")


@pytest.mark.parametrize("k", ["0", "3"])
@pytest.mark.parametrize("dtype", ["f32", "f16", "int8_rowwise", "int8_rowwise_split"])
def test_long_bags(dev, monkeypatch, dtype, k):
    say(f"[parity] long bags {dtype} k={k}")
    monkeypatch.setenv("EB_BAGS_PER_WAVE", k)
    D = {"f32": 64, "f16": 128}.get(dtype, 128)
    tables = [_table(dev, dtype, 5000, D)]
    w = _custom(dev, tables, [np.array([5000, 0, 1, 63, 64, 65, 1000, 4097])])
    full_check(w, f"long {dtype}")


def test_no_indices_at_all(dev):
    say("[parity] N = 0")
    tables = [_table(dev, "f32", 10, 16), _table(dev, "int8_rowwise", 10, 32)]
    w = _custom(dev, tables, [np.zeros(5, np.int64), np.zeros(5, np.int64)])
    got = run_gpu(w)
    assert torch.equal(got.view(torch.int32), torch.zeros_like(got).view(torch.int32))


def test_one_bag_one_table(dev):
    say("[parity] B = 1, T = 1")
    w = _custom(dev, [_table(dev, "f16", 50, 32)], [np.array([7])])
    full_check(w, "B=1")


def test_deterministic_bits(dev):
    say("[parity] determinism")
    w = make_workload("c3b", dev, **REDUCED["c3b"])
    a = run_gpu(w)
    b = run_gpu(w)
    assert torch.equal(a.view(torch.int32), b.view(torch.int32))


def test_side_stream(dev):
    say("[parity] side stream")
    w = make_workload("c5", dev, **REDUCED["c5"])
    s = torch.cuda.Stream(device=dev)
    full_check(w, "side stream", stream=s)


# ----------------------------------------------------------------------------
# argument errors through the ABI (host-side: nothing is enqueued)


@pytest.mark.parametrize("long_len", ["0", "16"])
def test_threads_share_a_handle(dev, monkeypatch, long_len):
    # Host threads may call the lookup on one handle at once (ctypes releases
    # the GIL during the call): its tables and settings are fixed, and with
    # the long-bag pass (EB_LONG_BAG=16: most bags queued) each call enqueues
    # its lookup and pass under the handle's lock, so no pass takes another
    # call's queue.  Each thread writes its own output; every result equals a
    # single-threaded call.
    import threading

    monkeypatch.setenv("EB_LONG_BAG", long_len)
    monkeypatch.setenv("EB_LONG_SEG", "64")
    say(f"[parity] four host threads on one handle, EB_LONG_BAG={long_len}")
    w = make_workload("c2", dev, **REDUCED["c2"])
    ws = [w] + [make_workload("c2", dev, batch_seed=s, tables=w.tables, **REDUCED["c2"]) for s in (1, 2, 3)]
    with eb.eb_create_tables(w.tables) as h:
        ref = []
        for x in ws:
            o = torch.empty((x.batch, x.sum_dim), device=dev)
            eb.eb_forward(h, x.indices, x.offsets, x.weights, x.pooling, o)
            ref.append(o)
        torch.cuda.synchronize()
        outs = [[torch.full((x.batch, x.sum_dim), float("nan"), device=dev) for _ in range(20)] for x in ws]
        errors = []

        def work(i):
            try:
                x = ws[i]
                for o in outs[i]:
                    eb.eb_forward(h, x.indices, x.offsets, x.weights, x.pooling, o)
            except Exception as e:  # reported below
                errors.append(e)

        threads = [threading.Thread(target=work, args=(i,)) for i in range(len(ws))]
        for th in threads:
            th.start()
        for th in threads:
            th.join()
        torch.cuda.synchronize()
    assert not errors, errors
    for i in range(len(ws)):
        for o in outs[i]:
            assert torch.equal(o.view(torch.int32), ref[i].view(torch.int32))


def test_forward_argument_errors(dev):
    say("[parity] argument errors")
    w = _custom(dev, [_table(dev, "f32", 10, 16), _table(dev, "f16", 10, 16)], [np.array([1, 2]), np.array([0, 3])])
    out = torch.full((2, 32), 7.0, device=dev)
    with eb.eb_create_tables(w.tables) as h:
        def expect(status, **kw):
            args = dict(indices=w.indices, offsets=w.offsets, per_sample_weights=None, pooling="sum", out=out)
            args.update(kw)
            with pytest.raises(eb.EBError) as e:
                eb.eb_forward(h, **args)
            assert e.value.status == status, kw.keys()

        expect(eb.EB_ERR_DTYPE, offsets=w.offsets.int())
        expect(eb.EB_ERR_DTYPE, indices=w.indices.float(), offsets=w.offsets.float())
        expect(eb.EB_ERR_DTYPE, out=out.double())
        expect(eb.EB_ERR_SHAPE, offsets=w.offsets[:-1].contiguous())
        expect(eb.EB_ERR_SHAPE, out=out[:1].contiguous())
        expect(eb.EB_ERR_SHAPE, per_sample_weights=torch.ones(w.num_indices + 1, device=dev))
        expect(eb.EB_ERR_INVALID_ARG, per_sample_weights=torch.ones(w.num_indices, device=dev), pooling="mean")
        expect(eb.EB_ERR_INVALID_ARG, pooling=5)
        expect(eb.EB_ERR_UNSUPPORTED, out=torch.empty(2 * 32 + 1, device=dev)[1:])
        torch.cuda.synchronize()
        assert torch.all(out == 7.0)  # nothing was written


def test_create_refuses_memory_the_gpu_cannot_read(dev):
    # kernels read the rows in place: pageable host memory is refused at
    # creation; device and pinned host memory are accepted (no lookup is run
    # on the host rows)
    say("[parity] table memory the GPU cannot read")
    import ctypes

    lib = eb.load_library()

    def create(ptr):
        arr = (eb.eb_table_desc * 1)(eb.eb_table_desc(ptr, 10, 16, eb.EB_F32, 64))
        h = ctypes.c_void_p(0)
        st = lib.eb_create_tables(arr, 1, None, ctypes.byref(h))
        return st, h.value

    host = np.zeros(10 * 16 + 4, np.float32)
    st, h = create((host.ctypes.data + 15) // 16 * 16)
    assert st == eb.EB_ERR_INVALID_ARG and h is None
    for rows in (torch.zeros((10, 16), device=dev), torch.zeros((10, 16), pin_memory=True)):
        st, h = create(rows.data_ptr())
        assert st == eb.EB_OK and h
        assert lib.eb_destroy(h) == eb.EB_OK
    with pytest.raises(ValueError):
        eb.eb_create_tables([(torch.zeros(10, 16), 16, "f32")])


def test_create_reports_out_of_memory(dev, monkeypatch):
    # a cap on the handle's device memory below what it needs: EB_ERR_OOM,
    # *out set to NULL, nothing leaked; a cap above it: a working handle
    say("[parity] device allocation refused at create time")
    import ctypes

    lib = eb.load_library()
    rows = torch.zeros((10, 16), device=dev)

    def create():
        arr = (eb.eb_table_desc * 1)(eb.eb_table_desc(rows.data_ptr(), 10, 16, eb.EB_F32, 64))
        h = ctypes.c_void_p(0xDEAD)  # must be overwritten
        st = lib.eb_create_tables(arr, 1, None, ctypes.byref(h))
        return st, h.value

    for cap in ("0", "1", "4096"):
        monkeypatch.setenv("EB_DEVICE_ALLOC_LIMIT", cap)
        st, h = create()
        assert st == eb.EB_ERR_OOM and h is None, (cap, st, h)
    monkeypatch.setenv("EB_DEVICE_ALLOC_LIMIT", str(1 << 22))
    st, h = create()
    assert st == eb.EB_OK and h
    out = torch.full((1, 16), float("nan"), device=dev)
    rows.copy_(torch.arange(160, dtype=torch.float32, device=dev).view(10, 16))
    idx, off = torch.tensor([3], device=dev), torch.tensor([0, 1], device=dev)  # kept alive past the call
    o, i, f = eb._as_tensor(out), eb._as_tensor(idx), eb._as_tensor(off)
    assert lib.eb_forward(h, i, f, eb._as_tensor(None), eb.EB_POOL_SUM, o) == eb.EB_OK
    assert lib.eb_destroy(h) == eb.EB_OK
    torch.cuda.synchronize()
    assert torch.equal(out[0], rows[3])


def test_checked_mode_reports_bad_data(dev, monkeypatch):
    say("[parity] checked mode")
    monkeypatch.setenv("EB_CHECK", "1")
    tb = _table(dev, "f32", 10, 16)
    out = torch.empty((3, 16), device=dev)
    with eb.eb_create_tables([tb]) as h:
        ok_idx = torch.tensor([1, 2, 3, 4], device=dev)
        off = torch.tensor([0, 2, 2, 4], device=dev)
        eb.eb_forward(h, ok_idx, off, None, "sum", out)  # valid: no error
        for bad_idx in ([1, 10, 3, 4], [1, -1, 3, 4]):  # the kernel skips such rows, never reads them
            with pytest.raises(eb.EBError) as e:
                eb.eb_forward(h, torch.tensor(bad_idx, device=dev), off, None, "sum", out)
            assert e.value.status == eb.EB_ERR_INDEX_OOB
        for bad_off in ([1, 2, 2, 4], [0, 3, 2, 4], [0, 2, 2, 3], [0, 2, 2, 9]):  # clamped in the kernel
            with pytest.raises(eb.EBError) as e:
                eb.eb_forward(h, ok_idx, torch.tensor(bad_off, device=dev), None, "sum", out)
            assert e.value.status == eb.EB_ERR_OFFSETS
        eb.eb_forward(h, ok_idx, off, None, "sum", out)  # the error word was cleared
    ref = ebo_forward([OracleTable(tb.rows.cpu().numpy(), 16, "f32")], np.array([1, 2, 3, 4]), np.array([0, 2, 2, 4]))
    assert ulp_distance(out.cpu().numpy(), ref).max() <= 1


def test_checked_mode_through_the_long_bag_pass(dev, monkeypatch):
    # bags of 40 lookups with EB_LONG_BAG=8, so every bag goes through the
    # pass (segments of 64 positions): an index outside the table inside a
    # long bag, and offsets that break the partition, are reported by
    # checked mode; a good call after them pools correctly
    say("[parity] checked mode through the long-bag pass")
    monkeypatch.setenv("EB_CHECK", "1")
    monkeypatch.setenv("EB_LONG_BAG", "8")
    monkeypatch.setenv("EB_LONG_SEG", "64")
    tb = _table(dev, "f32", 1000, 16)
    w = _custom(dev, [tb], [np.array([40, 40, 40])], seed=9)
    idx, off = w.indices, w.offsets
    out = torch.empty((3, 16), device=dev)
    with eb.eb_create_tables([tb]) as h:
        for where, bad in ((45, 1000), (100, -3)):
            b = idx.clone()
            b[where] = bad
            with pytest.raises(eb.EBError) as e:
                eb.eb_forward(h, b, off, None, "sum", out)
            assert e.value.status == eb.EB_ERR_INDEX_OOB
        for bad_off in ([0, 40, 30, 120], [0, 40, 80, 130]):
            with pytest.raises(eb.EBError) as e:
                eb.eb_forward(h, idx, torch.tensor(bad_off, device=dev), None, "sum", out)
            assert e.value.status == eb.EB_ERR_OFFSETS
        eb.eb_forward(h, idx, off, None, "sum", out)
    tabs = oracle_tables(w)
    ref, asum = oracle_forward(w, tables=tabs)
    check(out.cpu().numpy(), ref, asum, per_element_lengths(w), RTOL["f32"], "checked long pass",
          split_scale(w, tabs))


@pytest.mark.parametrize("index_dtype", [torch.int32, torch.int64])
def test_long_bag_pass_index_types(dev, monkeypatch, index_dtype):
    # the pass stages 32- and 64-bit indices alike (widened to 64 bits in LDS)
    say(f"[parity] long-bag pass, {index_dtype} indices")
    monkeypatch.setenv("EB_LONG_BAG", "32")
    monkeypatch.setenv("EB_LONG_SEG", "64")
    rng = np.random.default_rng(33)
    tables = [_table(dev, "f16", 3000, 128), _table(dev, "int8_rowwise", 2000, 64, seed=1)]
    lens = [rng.integers(0, 400, 40) for _ in tables]
    w = _custom(dev, tables, lens, weighted=True, index_dtype=index_dtype)
    full_check(w, f"long pass {index_dtype}")


@pytest.mark.parametrize("case", range(12))
def test_long_bag_pass_random_settings(dev, monkeypatch, case):
    # seeded random mixes through the pass: two to four tables of any storage
    # type and width, long-tailed bag lengths up to a few thousand, every
    # pooling mode and index width, thresholds from 4 to 512 and segments
    # from 64 to 2048 positions
    rng = np.random.default_rng(700 + case)
    dtypes = ["f32", "f16", "int8_rowwise", "int8_rowwise_split"]
    nt = int(rng.integers(2, 5))
    tables = []
    for t in range(nt):
        dt = dtypes[int(rng.integers(0, 4))]
        mult = {"f32": 4, "f16": 8, "int8_rowwise": 16, "int8_rowwise_split": 16}[dt]
        D = mult * int(rng.integers(1, 33))
        tables.append(_table(dev, dt, int(rng.integers(50, 5000)), D, seed=case * 10 + t))
    B = int(rng.integers(1, 60))
    lens = [np.minimum(rng.lognormal(3.0, 1.6, B).astype(np.int64), 6000) for _ in tables]
    mode = ["sum", "mean", "weighted"][case % 3]
    long_len = str(int(rng.choice([4, 16, 64, 200, 512])))
    seg = str(int(rng.choice([64, 128, 512, 2048])))
    idt = torch.int32 if case % 4 == 1 else torch.int64
    say(f"[parity] long-bag pass random case {case}: {nt} tables, B={B}, {mode}, long>{long_len}, seg {seg}, "
        f"{idt}, longest {max(int(l.max()) for l in lens)}")
    monkeypatch.setenv("EB_LONG_BAG", long_len)
    monkeypatch.setenv("EB_LONG_SEG", seg)
    w = _custom(dev, tables, lens, weighted=(mode == "weighted"), pooling="mean" if mode == "mean" else "sum",
                index_dtype=idt, seed=case)
    got = full_check(w, f"random case {case}")
    # deterministic: the same call again gives the same bits
    assert np.array_equal(got.view(np.uint32), run_gpu(w).cpu().numpy().view(np.uint32)), case


def test_native_library_is_the_one_loaded(dev):
    lib = eb.load_library()
    assert os.path.samefile(lib._name, eb.LIB_PATH)
