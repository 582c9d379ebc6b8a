import os
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (runs through the libeb C ABI)")


# ----------------------------------------------------------------------------
# shared helpers (plain numpy; no pooling arithmetic lives here)


def ulp_distance(a, b):
    """Distance in units in the last place between fp32 arrays (0 = same bits,
    except +0 and -0 count as 0 apart)."""
    a = np.ascontiguousarray(a, dtype=np.float32).view(np.int32).astype(np.int64)
    b = np.ascontiguousarray(b, dtype=np.float32).view(np.int32).astype(np.int64)
    # map the sign-magnitude bit patterns onto a monotone integer line
    a = np.where(a < 0, -(a & 0x7FFFFFFF), a)
    b = np.where(b < 0, -(b & 0x7FFFFFFF), b)
    return np.abs(a - b)


def oracle_tables(workload):
    """Host copies of a workload's tables in the oracle's format."""
    from oracle import OracleTable

    return [OracleTable.of(t) for t in workload.tables]


def compact_oracle_table(tb, rows):
    """An OracleTable holding only rows `rows` (in that order, renumbered
    0..len-1) of a workload Table, in the table's own layout.  Data movement
    only."""
    import torch
    from oracle import OracleTable

    rows = np.asarray(rows, np.int64)
    sel = torch.from_numpy(rows if rows.size else np.zeros(1, np.int64)).to(tb.rows.device)
    if tb.dtype == "int8_rowwise_split":
        R, st = tb.num_rows, tb.row_stride_bytes
        codes = tb.rows.index_select(0, sel)
        words = tb.storage[R * st:R * st + 4 * R].view(R, 4).index_select(0, sel)
        buf = torch.cat([codes.reshape(-1), words.reshape(-1)]).cpu().numpy()
        return OracleTable(buf, tb.dim, tb.dtype, int(sel.numel()), st)
    return OracleTable(np.ascontiguousarray(tb.rows.index_select(0, sel).cpu().numpy()), tb.dim, tb.dtype)


def oracle_forward(workload, tables=None, bags=None, with_absum=True, num_threads=0):
    from oracle import ebo_forward

    tables = oracle_tables(workload) if tables is None else tables
    w = None if workload.weights is None else workload.weights.cpu().numpy()
    return ebo_forward(tables, workload.indices.cpu().numpy(), workload.offsets.cpu().numpy(), w,
                       workload.pooling, bags=bags, num_threads=num_threads, with_absum=with_absum)


@pytest.fixture(scope="session", autouse=True)
def _build_oracle_once():
    from oracle import build, lib_path

    src = os.path.join(ROOT, "oracle", "eb_oracle.c")
    if os.environ.get("EBO_ORACLE_LIB"):
        pass  # another build of the oracle (the sanitizer run) is loaded as given
    elif not os.path.exists(lib_path()) or os.path.getmtime(lib_path()) < os.path.getmtime(src):
        build()
    yield
