"""Write oracle_regression.json: a frozen record of the oracle on small inputs.

Calls only the oracle (and numpy for seeded inputs).  The fixture lets a test
detect any later change in the oracle's arithmetic; such a change must come
with a new fixture and, in its commit message, the passage or reading of the
paper that justifies it.  It records the pooled lookup of the paper's
sparse_arch stage (Sec. IV-A.2) over jagged categorical features (Abstract),
the un-pooled lookup, the FM cross term over the pooled fields (inter_arch.fm,
Sec. IV-A.2), and the backward with a row-wise optimizer step (Sec. III-A).

    python tests/golden/make_golden.py
"""
import json
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from oracle import OracleTable, ebo_backward_update, ebo_fm, ebo_forward, ebo_forward_seq  # noqa: E402


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


def backward_cases(tables, idx, off, w):
    """SGD and row-wise Adagrad on the fp32 and fp16 tables (the first two
    tables' bags of the lookup cases), one seeded output gradient."""
    T, B = 3, (off.size - 1) // 3
    n2 = int(off[2 * B])
    off2 = off[:2 * B + 1]
    idx2 = idx[:n2]
    grad = np.random.default_rng([2609, 98]).standard_normal((B, 16)).astype(np.float32)
    for opt, mode, weights in (("sgd", "sum", None), ("rowwise_adagrad", "mean", None),
                               ("rowwise_adagrad", "sum", None if w is None else w[:n2])):
        tabs = [OracleTable(tables["f32"].copy(), 8, "f32"), OracleTable(tables["f16"].copy(), 8, "f16")]
        state = np.linspace(0.0, 1.0, 24).astype(np.float32)
        ebo_backward_update(tabs, idx2, off2, weights, mode, grad, opt, lr=0.05, eps=1e-3, state=state)
        yield {
            "offsets": off2.tolist(), "indices": idx2.tolist(), "pooling": mode, "optimizer": opt,
            "weights": None if weights is None else weights.view(np.uint32).tolist(),
            "grad_bits": grad.view(np.uint32).tolist(), "lr": 0.05, "eps": 1e-3,
            "state_in_bits": np.linspace(0.0, 1.0, 24).astype(np.float32).view(np.uint32).tolist(),
            "f32_bits": tabs[0].rows.view(np.uint32).tolist(), "f16_bits": tabs[1].rows.view(np.uint16).tolist(),
            "state_bits": state.view(np.uint32).tolist(),
        }


def main():
    out = []
    train = []
    for tables, idx, off, w, mode in cases():
        tabs = [OracleTable(tables[k], 8, k) for k in ("f32", "f16", "int8_rowwise")]
        res = ebo_forward(tabs, idx, off, w, mode)
        seq = ebo_forward_seq(tabs, idx, off)
        fm = ebo_fm(res, 3, 8)
        out.append({
            "tables": {k: v.view(np.uint8).reshape(v.shape[0], -1).tolist() for k, v in tables.items()},
            "dim": 8,
            "indices": idx.tolist(),
            "offsets": off.tolist(),
            "weights": None if w is None else w.view(np.uint32).tolist(),
            "pooling": mode,
            "out_bits": res.view(np.uint32).tolist(),
            "seq_bits": seq.view(np.uint32).tolist(),
            "fm_bits": [int(x) for x in fm.view(np.uint64)],
        })
        if mode == "sum" and w is not None:
            train = list(backward_cases(tables, idx, off, w))
    doc = {
        "about": "oracle outputs (bit patterns) on three tables f32/f16/int8_rowwise (D=8, 12 rows), B=6, "
                 "written by tests/golden/make_golden.py: pooled lookup of sparse_arch (Sec. IV-A.2; fp32), "
                 "un-pooled lookup (fp32), FM cross term over the three pooled fields (fp64), and the backward "
                 "with SGD / row-wise Adagrad on the fp32 and fp16 tables (Sec. III-A)",
        "cases": out,
        "backward": train,
    }
    with open(os.path.join(HERE, "oracle_regression.json"), "w") as f:
        json.dump(doc, f)


if __name__ == "__main__":
    main()
