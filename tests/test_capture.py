"""Top-P capture of the tiled (App. B) and exact importance on synthetic keys.

The paper's tiled-capture table compares the fraction of true attention mass
that falls on the keys of the selected parents when the selection comes from
the tiled importance (count-extrapolated denominator), from the exact
importance, and from the best possible choice (the P parents whose keys get
the most true mass). This test computes the same three numbers with the
oracle on a synthetic workload of the table's shape (M0 = 256, Ch = 8,
P in {24, 32}, codeword tiles of 128 parents as in the paper and of 64 as in
the kernel) and checks what holds whatever the data: no selection beats the
best one. Run with ``-s`` to print the table.
"""
import numpy as np
import pytest

import oracle
from paper_2607_12789_amd import inputs

W = inputs.Workload("capture", B=1, H=2, N=2048, d=64, M0=256, Ch=8, P=32, block_q=128,
                    dtype="f32", q_scale=6.0, dirichlet_alpha=0.5, seed=11)


@pytest.fixture(scope="module")
def setup():
    x = inputs.generate(W)
    a = oracle.assign(x["K"], x["Cp"], x["Cc"])
    _, counts = oracle.aggregate(x["V"], a["parent_idx"], a["code_idx"], W.M0, W.Ch)
    exact = oracle.importance(x["Q"], x["Cp"], counts, W.Ch, W.block_q)
    tiled = {tc: oracle.importance_tiled(x["Q"], x["Cp"], counts, W.Ch, W.block_q, tc)
             for tc in (64, 128)}
    return x, a, exact, tiled


@pytest.mark.parametrize("P", [24, 32])
def test_capture_table(setup, P):
    x, a, exact, tiled = setup
    rows = {"non-tiled": oracle.topp(exact, P)}
    rows.update({f"tiled {tc}": oracle.topp(w, P) for tc, w in tiled.items()})
    best = None
    for name, sel in rows.items():
        cap = oracle.capture(x["Q"], x["K"], a["parent_idx"], sel, W.block_q)
        best = cap["exact"] if best is None else best
        assert abs(cap["exact"] - best) < 1e-12
        assert 0.0 < cap["selected"] <= cap["exact"] + 1e-12
        print(f"P={P} {name:10s} capture {100 * cap['selected']:.1f}%")
    print(f"P={P} exact      capture {100 * best:.1f}%")
    # the tiled selections differ from the exact-importance one somewhere
    assert any((rows[k] != rows["non-tiled"]).any() for k in rows if k != "non-tiled")
