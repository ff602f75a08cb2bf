"""The Gilbert token order (avq_gilbert_order, host code) and what it is for.

Pins: every grid from 1x1 to 40x40 gets a permutation of its cells that
starts at (0, 0), moves to a 4-neighbour at every step except for at most one
diagonal step; on 2^k x 2^k grids it is, up to one of the 8 symmetries of the
square, the Hilbert curve of the textbook index-to-cell conversion; runs of
consecutive tokens are compact. Then the reason for the order (Sec. 4,
App. spatial reordering ablation): on spatially structured tokens, tiles of
consecutive tokens along the curve capture more attention mass with their
top-P parents than raster strips, and both beat a random order (the oracle's
capture metric).
"""
import numpy as np
import pytest

import oracle
from paper_2607_12789_amd import avq, inputs
from tests import references as ref

OK, INVALID, UNSUPPORTED = avq.AVQ_OK, avq.AVQ_ERR_INVALID_ARG, avq.AVQ_ERR_UNSUPPORTED


def cells(order, width):
    o = np.asarray(order, dtype=np.int64)
    return o % width, o // width


def test_every_grid_gets_a_curve():
    for width in range(1, 41):
        for height in range(1, 41):
            order, rank = avq.gilbert_order(width, height)
            o = order.numpy()
            assert sorted(o.tolist()) == list(range(width * height)), (width, height)
            np.testing.assert_array_equal(rank.numpy()[o], np.arange(width * height))
            x, y = cells(o, width)
            assert x[0] == 0 and y[0] == 0
            dx, dy = np.abs(np.diff(x)), np.abs(np.diff(y))
            steps = dx + dy
            diag = (dx == 1) & (dy == 1)
            assert ((steps == 1) | diag).all(), (width, height)
            assert diag.sum() <= 1, (width, height)


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5])
def test_power_of_two_square_is_a_hilbert_curve(k):
    n = 1 << k
    hx, hy = ref.hilbert_cells(n)
    order, _ = avq.gilbert_order(n, n)
    x, y = cells(order.numpy(), n)
    found = False
    for sx in (False, True):
        for sy in (False, True):
            for swap in (False, True):
                a, b = (hy, hx) if swap else (hx, hy)
                a = n - 1 - a if sx else a
                b = n - 1 - b if sy else b
                found |= bool((a == x).all() and (b == y).all())
    assert found


def test_runs_are_compact():
    """Runs of 64 consecutive tokens stay compact: the longer side of their
    bounding box averages at most 12 cells on the 28x28 patch grid of the
    paper's figure and on 128x128 (a raster run spans 28 and 64 cells)."""
    for width, height in ((28, 28), (128, 128)):
        order, _ = avq.gilbert_order(width, height)
        x, y = cells(order.numpy(), width)
        n = width * height
        ext = []
        for t in range(0, n - 63, 64):
            xs, ys = x[t:t + 64], y[t:t + 64]
            ext.append(max(xs.max() - xs.min() + 1, ys.max() - ys.min() + 1))
        assert np.mean(ext) <= 12, (width, height, np.mean(ext))


def test_gilbert_order_validation():
    L = avq.lib()
    import ctypes
    buf = (ctypes.c_int32 * 4)()
    assert L.avq_gilbert_order(0, 3, buf, None) == INVALID
    assert L.avq_gilbert_order(2, 2, None, None) == INVALID
    assert L.avq_gilbert_order(1 << 13, 1 << 12, buf, None) == UNSUPPORTED
    assert L.avq_gilbert_order(2, 2, buf, None) == OK
    assert sorted(buf) == [0, 1, 2, 3]


W = inputs.Workload("spatial", B=1, H=2, N=4096, d=64, M0=64, Ch=8, P=16, block_q=64,
                    dtype="f32", q_scale=8.0, seed=3)


@pytest.fixture(scope="module")
def spatial_setup():
    x = inputs.spatial(W, 64, 64)
    a = oracle.assign(x["K"], x["Cp"], x["Cc"])
    _, counts = oracle.aggregate(x["V"], a["parent_idx"], a["code_idx"], W.M0, W.Ch)
    return x, a, counts


@pytest.mark.parametrize("block_q", [32, 64, 128])
def test_curve_order_captures_more(spatial_setup, block_q):
    """The synthetic counterpart of the reordering ablation (M0 = 64, P = 16,
    Ch = 8, tiles of 32, 64, 128): capture of the top-P selection per tile."""
    x, a, counts = spatial_setup
    orders = {"gilbert": avq.gilbert_order(64, 64)[0].numpy(),
              "raster": np.arange(W.N),
              "random": np.random.default_rng(0).permutation(W.N)}
    cap = {}
    for name, o in orders.items():
        Qp = x["Q"][:, :, o]
        sel = oracle.topp(oracle.importance(Qp, x["Cp"], counts, W.Ch, block_q), W.P)
        cap[name] = oracle.capture(Qp, x["K"], a["parent_idx"], sel, block_q)["selected"]
    print(f"block_q={block_q}: " + ", ".join(f"{k} {100 * v:.1f}%" for k, v in cap.items()))
    assert cap["gilbert"] >= cap["raster"] - 0.005
    assert cap["raster"] > cap["random"] + 0.05
