"""Write oracle_regression.json: a frozen record of the oracle on small inputs.

Calls only the oracle (and numpy for seeded inputs).  The fixture lets a test
detect any later change in the oracle's arithmetic; such a change must come
with a new fixture and, in its commit message, the passage or reading of the
paper that justifies it.  The pooled lookup it records is the paper's
sparse_arch stage (Sec. IV-A.2) over jagged categorical features (Abstract).

    python tests/golden/make_golden.py
"""
import json
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from oracle import OracleTable, ebo_forward  # noqa: E402


def cases():
    rng = np.random.default_rng([2609, 99])
    R, D, B = 12, 8, 6
    f32 = rng.uniform(-1, 1, (R, D)).astype(np.float32)
    f16 = (rng.standard_normal((R, D)) * 0.01).astype(np.float16)
    u8 = np.zeros((R, D + 4), np.uint8)
    u8[:, :D] = rng.integers(0, 256, (R, D))
    u8[:, D:D + 2] = rng.uniform(1e-4, 4e-4, R).astype(np.float16).view(np.uint8).reshape(R, 2)
    u8[:, D + 2:] = rng.uniform(-0.06, -0.02, R).astype(np.float16).view(np.uint8).reshape(R, 2)
    lens = rng.integers(0, 7, 3 * B)
    off = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    idx = rng.integers(0, R, off[-1]).astype(np.int64)
    w = rng.uniform(0, 1, off[-1]).astype(np.float32)
    tables = {"f32": f32, "f16": f16, "int8_rowwise": u8}
    for mode, weights in (("sum", None), ("mean", None), ("sum", w)):
        yield tables, idx, off, weights, mode


def main():
    out = []
    for tables, idx, off, w, mode in cases():
        tabs = [OracleTable(tables[k], 8, k) for k in ("f32", "f16", "int8_rowwise")]
        res = ebo_forward(tabs, idx, off, w, mode)
        out.append({
            "tables": {k: v.view(np.uint8).reshape(v.shape[0], -1).tolist() for k, v in tables.items()},
            "dim": 8,
            "indices": idx.tolist(),
            "offsets": off.tolist(),
            "weights": None if w is None else w.view(np.uint32).tolist(),
            "pooling": mode,
            "out_bits": res.view(np.uint32).tolist(),
        })
    doc = {
        "about": "oracle outputs (fp32 bit patterns) on three tables f32/f16/int8_rowwise (D=8, 12 rows), "
                 "B=6, written by tests/golden/make_golden.py; pooled lookup of sparse_arch, Sec. IV-A.2",
        "cases": out,
    }
    with open(os.path.join(HERE, "oracle_regression.json"), "w") as f:
        json.dump(doc, f)


if __name__ == "__main__":
    main()
