"""The lookups and the backward under HIP graph capture: eb_forward (the
lookup and its long-bag pass), eb_forward_fm, eb_forward_seq and the
backward (given a workspace, or its no-allocation entry point) allocate
nothing and (outside checked mode) enqueue only kernels on the handle's
stream, so a caller can capture them once and replay them (on the handle's
stream, or ordered with it: the long-bag pass keeps a queue in the handle).
Each test captures one call on the handle's stream, then replays it
several times, with eager work of the program and synchronisations between the
replays and new index contents copied into the captured buffers, and checks
every replay bit for bit against an eager call on the same inputs (the kernels
are deterministic).
"""
import pytest
import torch

from paper_2609_30656_amd import eb
from paper_2609_30656_amd.workload import make_workload

pytestmark = pytest.mark.gpu

SMALL = {
    "c2": dict(rows_cap=20000, batch=256),
    "c3b": dict(rows_cap=50000, batch=256),
    "c5": dict(rows_cap=20000, batch=128),
}


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


def _batches(name, dev):
    """Two index batches of one workload over the same tables, with the same
    number of lookups (the second batch's indices permuted within each
    table), so both fit the captured buffers."""
    w = make_workload(name, dev, **SMALL[name])
    off = w.offsets.cpu()
    idx2 = w.indices.clone()
    g = torch.Generator(device="cpu")
    g.manual_seed(3)
    for t in range(w.num_tables):
        lo, hi = int(off[t * w.batch]), int(off[(t + 1) * w.batch])
        idx2[lo:hi] = w.indices[lo:hi][torch.randperm(hi - lo, generator=g).to(dev)]
    return w, idx2


def _replay_and_check(run_into, fresh_outputs, w, idx2, stream, label):
    """run_into(outs) enqueues the call writing into outs (a tuple of tensors)."""
    idx_buf = w.indices.clone()
    captured = fresh_outputs()
    # warm the call up on the capture stream before capturing, as torch asks
    with torch.cuda.stream(stream):
        run_into(idx_buf, captured)
    stream.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=stream):
        run_into(idx_buf, captured)
    for rep, src in enumerate([w.indices, idx2, w.indices, idx2]):
        idx_buf.copy_(src)
        torch.cuda.synchronize()
        for o in captured:
            o.fill_(float("nan"))  # the replay must write every element
        with torch.cuda.stream(stream):  # on the handle's stream, as its calls go
            graph.replay()
        # eager work of the program between replays
        eager = fresh_outputs()
        with torch.cuda.stream(stream):
            run_into(src, eager)
        junk = torch.randn(1 << 20, device=w.indices.device).sum()
        torch.cuda.synchronize()
        for a, b in zip(captured, eager):
            assert torch.equal(a.view(torch.int32), b.view(torch.int32)), f"{label}: replay {rep} differs"
        assert torch.isfinite(junk)
    del graph


@pytest.mark.parametrize("name", list(SMALL))
def test_forward_replays(dev, name):
    say(f"[graph] eb_forward {name}")
    w, idx2 = _batches(name, dev)
    stream = torch.cuda.Stream(device=dev)
    with eb.eb_create_tables(w.tables, stream) as h:
        def run_into(idx, outs):
            eb.eb_forward(h, idx, w.offsets, w.weights, w.pooling, outs[0])

        def fresh():
            return (torch.empty((w.batch, w.sum_dim), device=dev),)

        _replay_and_check(run_into, fresh, w, idx2, stream, f"forward {name}")


@pytest.mark.parametrize("name", ["c2", "c5"])
def test_forward_fm_replays(dev, name):
    say(f"[graph] eb_forward_fm {name}")
    w, idx2 = _batches(name, dev)
    stream = torch.cuda.Stream(device=dev)
    with eb.eb_create_tables(w.tables, stream) as h:
        def run_into(idx, outs):
            eb.eb_forward_fm(h, idx, w.offsets, w.weights, w.pooling, outs[0], outs[1])

        def fresh():
            return torch.empty((w.batch, w.sum_dim), device=dev), torch.empty(w.batch, device=dev)

        _replay_and_check(run_into, fresh, w, idx2, stream, f"forward_fm {name}")


@pytest.mark.parametrize("name", ["c2", "c5"])
def test_sequence_lookup_replays(dev, name):
    say(f"[graph] eb_forward_seq {name}")
    w, idx2 = _batches(name, dev)
    stream = torch.cuda.Stream(device=dev)
    with eb.eb_create_tables(w.tables, stream) as h:
        def run_into(idx, outs):
            eb.eb_forward_seq(h, idx, w.offsets, outs[0])

        def fresh():
            return (torch.empty(w.seq_output_numel(), device=dev),)

        _replay_and_check(run_into, fresh, w, idx2, stream, f"seq {name}")


@pytest.mark.parametrize("name", ["c3b", "c5"])
def test_forward_replays_with_long_bags(dev, monkeypatch, name):
    # most bags left to the long-bag pass (a second kernel, with a queue and
    # counters in the handle): each replay must find the counters cleared by
    # the previous call, captured or eager
    say(f"[graph] eb_forward {name}, long-bag pass")
    monkeypatch.setenv("EB_LONG_BAG", "16")
    monkeypatch.setenv("EB_LONG_SEG", "64")
    w, idx2 = _batches(name, dev)
    stream = torch.cuda.Stream(device=dev)
    with eb.eb_create_tables(w.tables, stream) as h:
        def run_into(idx, outs):
            eb.eb_forward(h, idx, w.offsets, w.weights, w.pooling, outs[0])

        def fresh():
            return (torch.empty((w.batch, w.sum_dim), device=dev),)

        _replay_and_check(run_into, fresh, w, idx2, stream, f"forward long {name}")


def _clone_tables(tables):
    from paper_2609_30656_amd.workload import Table
    return [Table(t.rows.clone(), t.dim, t.dtype) for t in tables]


@pytest.mark.parametrize("name,entry", [("c2", "workspace"), ("c3b", "workspace"), ("c2", "noalloc")])
def test_backward_replays(dev, name, entry):
    """The backward with row-wise Adagrad under capture: outside checked mode
    eb_backward_update (given a workspace) and eb_backward_update_noalloc
    enqueue only kernels, and its sort clears its own counters with a kernel.
    Replays of a captured step, fed new indices and gradients through the
    captured buffers, must leave the tables and the optimizer state bit for
    bit where the same eager calls on a copy leave them."""
    say(f"[graph] backward {name} {entry}")
    w, idx2 = _batches(name, dev)
    stream = torch.cuda.Stream(device=dev)
    tabs_g, tabs_e = _clone_tables(w.tables), _clone_tables(w.tables)
    R = sum(t.num_rows for t in w.tables)
    g = torch.Generator(device=dev)
    g.manual_seed(5)
    st_g = torch.rand(R, generator=g, device=dev)
    st_e = st_g.clone()
    grads = [torch.randn((w.batch, w.sum_dim), generator=g, device=dev) for _ in range(5)]
    idx_buf, grad_buf = w.indices.clone(), grads[0].clone()
    with eb.eb_create_tables(tabs_g, stream) as hg, eb.eb_create_tables(tabs_e, stream) as he:
        ws = torch.empty(eb.eb_backward_workspace_size(hg, w.num_indices), dtype=torch.uint8, device=dev)
        ws_e = torch.empty_like(ws)

        def step(h, idx, grad, st, workspace):
            if entry == "noalloc":
                eb.eb_backward_update_noalloc(h, idx, w.offsets, w.weights, w.pooling, grad, "rowwise_adagrad",
                                              0.05, 1e-4, st)
            else:
                eb.eb_backward_update(h, idx, w.offsets, w.weights, w.pooling, grad, "rowwise_adagrad", 0.05,
                                      1e-4, st, workspace=workspace)

        # warm-up on the capture stream, matched by the same eager step on the copy
        with torch.cuda.stream(stream):
            step(hg, idx_buf, grad_buf, st_g, ws)
            step(he, w.indices, grads[0], st_e, ws_e)
        stream.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=stream):
            step(hg, idx_buf, grad_buf, st_g, ws)
        for rep, (src, grad) in enumerate(zip([w.indices, idx2, w.indices, idx2], grads[1:])):
            idx_buf.copy_(src)
            grad_buf.copy_(grad)
            torch.cuda.synchronize()
            with torch.cuda.stream(stream):
                graph.replay()
            torch.cuda.synchronize()
            with torch.cuda.stream(stream):
                step(he, src, grad, st_e, ws_e)
            junk = torch.randn(1 << 20, device=dev).sum()  # eager work of the program between replays
            torch.cuda.synchronize()
            for t, (a, b) in enumerate(zip(tabs_g, tabs_e)):
                assert torch.equal(a.rows.view(torch.uint8), b.rows.view(torch.uint8)), \
                    f"backward {name} {entry}: replay {rep} table {t} differs"
            assert torch.equal(st_g.view(torch.int32), st_e.view(torch.int32)), \
                f"backward {name} {entry}: replay {rep} optimizer state differs"
            assert torch.isfinite(junk)
        del graph
