"""eb_backward_update_noalloc against eb_backward_update, through the C ABI.

The no-allocation entry point runs the same kernels with the library's
static device workspace instead of the caller's.  The backward is
deterministic (no floating-point atomics, fixed summation order), so on the
same inputs both entry points must leave the tables and the optimizer state
bit for bit the same.  Two calls in a row, the second on a smaller batch,
check that what the first left in the static array does not leak into the
second; a batch that needs more workspace than the array holds is refused
before anything is enqueued.
"""
import ctypes

import numpy as np
import pytest
import torch

from paper_2609_30656_amd import eb
from paper_2609_30656_amd.workload import Table, make_workload

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


def _bits(t):
    return t.detach().cpu().numpy().view(np.uint16 if t.dtype == torch.float16 else np.uint32).copy()


def _clone_tables(tables):
    return [Table(t.rows.clone(), t.dim, t.dtype) for t in tables]


@pytest.mark.parametrize("name,optimizer", [("c2", "rowwise_adagrad"), ("c3b", "rowwise_adagrad"),
                                            ("c3a", "sgd")])
def test_noalloc_matches_workspace_entry_point(dev, name, optimizer):
    shapes = [dict(rows_cap=20000, batch=512), dict(rows_cap=20000, batch=96)]  # second call: a smaller batch
    base = make_workload(name, dev, **shapes[0])
    tabs_ws, tabs_na = _clone_tables(base.tables), _clone_tables(base.tables)
    R = sum(t.num_rows for t in base.tables)
    g = torch.Generator(device=dev)
    g.manual_seed(3)
    state0 = torch.rand(R, generator=g, device=dev, dtype=torch.float32)
    st_ws, st_na = state0.clone(), state0.clone()
    with eb.eb_create_tables(tabs_ws) as h_ws, eb.eb_create_tables(tabs_na) as h_na:
        for call, shape in enumerate(shapes):
            w = make_workload(name, dev, batch_seed=call, tables=base.tables, **shape)
            grad = torch.randn((w.batch, w.sum_dim), generator=g, device=dev, dtype=torch.float32)
            need = eb.eb_backward_workspace_size(h_na, w.num_indices)
            say(f"[noalloc] {name} call {call}: {w.num_indices} lookups, batch {w.batch}, workspace {need} B")
            assert need <= eb.EB_NOALLOC_SCRATCH_BYTES
            before = [_bits(t.rows) for t in tabs_na]
            eb.eb_backward_update(h_ws, w.indices, w.offsets, w.weights, w.pooling, grad, optimizer, 0.05, 1e-4,
                                  st_ws)
            eb.eb_backward_update_noalloc(h_na, w.indices, w.offsets, w.weights, w.pooling, grad, optimizer, 0.05,
                                          1e-4, st_na)
            torch.cuda.synchronize()
            changed = 0
            for t, (a, b) in enumerate(zip(tabs_ws, tabs_na)):
                ba, bb = _bits(a.rows), _bits(b.rows)
                assert np.array_equal(ba, bb), f"{name} call {call} table {t}: {np.count_nonzero(ba != bb)} differ"
                changed += np.count_nonzero(bb != before[t])
            assert changed > 0, "the step updated nothing"
            assert np.array_equal(_bits(st_ws), _bits(st_na)), f"{name} call {call}: optimizer state differs"


def test_noalloc_refuses_a_batch_past_its_workspace(dev):
    # 4 M lookups into a 256-wide fp32 table need more than the static
    # workspace holds: refused on the host, nothing enqueued or written
    say("[noalloc] oversized batch")
    rows = torch.randn((1000, 256), device=dev)
    before = rows.clone()
    n = 4 << 20
    idx = torch.randint(0, 1000, (n,), device=dev, dtype=torch.int32)
    off = torch.tensor([0, n], device=dev, dtype=torch.int32)
    grad = torch.ones((1, 256), device=dev)
    with eb.eb_create_tables([Table(rows, 256, "f32")]) as h:
        assert eb.eb_backward_workspace_size(h, n) > eb.EB_NOALLOC_SCRATCH_BYTES
        with pytest.raises(eb.EBError) as e:
            eb.eb_backward_update_noalloc(h, idx, off, None, "sum", grad, "sgd", 0.1)
        assert e.value.status == eb.EB_ERR_UNSUPPORTED
        torch.cuda.synchronize()
    assert torch.equal(rows, before)


def test_noalloc_argument_errors(dev):
    say("[noalloc] argument errors")
    lib = eb.load_library()
    none = eb._as_tensor(None)
    assert lib.eb_backward_update_noalloc(None, none, none, none, 0, none, 0, ctypes.c_float(0.1),
                                          ctypes.c_float(0.0), none) == eb.EB_ERR_INVALID_ARG
    rows = torch.zeros((10, 16), device=dev)
    with eb.eb_create_tables([Table(rows, 16, "f32")]) as h:
        idx = torch.tensor([1, 2], device=dev)
        off = torch.tensor([0, 2], device=dev)
        with pytest.raises(eb.EBError) as e:  # Adagrad without its state
            eb.eb_backward_update_noalloc(h, idx, off, None, "sum", torch.ones((1, 16), device=dev),
                                          "rowwise_adagrad", 0.1)
        assert e.value.status == eb.EB_ERR_INVALID_ARG
        with pytest.raises(eb.EBError) as e:  # grad of the wrong size
            eb.eb_backward_update_noalloc(h, idx, off, None, "sum", torch.ones((2, 16), device=dev), "sgd", 0.1)
        assert e.value.status == eb.EB_ERR_SHAPE
        # no lookups: nothing to do
        eb.eb_backward_update_noalloc(h, idx[:0], torch.tensor([0, 0], device=dev), None, "sum",
                                      torch.ones((1, 16), device=dev), "sgd", 0.1)
        torch.cuda.synchronize()
    assert torch.count_nonzero(rows) == 0
