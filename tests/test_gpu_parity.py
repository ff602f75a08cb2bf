"""Parity of the HIP path (through the C ABI) with the fp64 oracle.

Every case draws seeded inputs, runs the precompute (avq_assign_aggregate,
or avq_assign -> avq_aggregate) and avq_attention_fwd on the GPU and the
oracle on the CPU, and compares (see tests/parity.py): assignments, counts and top-P sets exactly on certified
decisions, Vbar within the fp32 summation bound, importance within eps_w,
and Y per row within 1e-4 (fp32) / 2e-2 (bf16) relative to max|Y*|.

The five evaluation workloads run at their full sizes in the same launch
configuration as the benchmark, every query tile of every head compared.
"""
import sys

import numpy as np
import pytest
import torch

from paper_2607_12789_amd import inputs
from tests import parity

pytestmark = pytest.mark.gpu


def banner(name, w):
    print(f"\n[case] {name}: {w.describe()}", flush=True)
    sys.stdout.flush()


def report(res):
    for k in ("assign", "aggregate", "topp", "output"):
        print(f"  {k}: {res[k].line()}", flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_12789_amd import avq
    avq.lib()


def small(**kw):
    base = dict(name="edge", B=2, H=3, N=1000, d=64, M0=40, Ch=4, P=5, block_q=128,
                dtype="bf16", sigma_c=0.1, sigma_k=0.05, q_scale=2.0, seed=1)
    base.update(kw)
    return inputs.Workload(**base)


EDGE = {
    "ragged_n": small(),
    "n_one": small(N=1, B=1, H=1),
    "n_17_bq16": small(N=17, block_q=16),
    "p_zero": small(P=0),
    "p_full": small(P=40),
    "m0_37_ch16_d128": small(M0=37, Ch=16, d=128, P=7),
    "ch1": small(Ch=1, P=3),
    "ch2": small(Ch=2, P=9),
    "ch8_bq200": small(Ch=8, block_q=200, N=1300, P=11),
    "keys_stay": small(sigma_k=0.2, Ch=8, P=6),
    "dirichlet_sparse": small(dirichlet_alpha=0.05, M0=64, Ch=8, P=20, N=2000),
    "large_logits": small(q_scale=40.0, Ch=8, P=6),
    "fp32_d128": small(dtype="f32", d=128, Ch=8, P=4, block_q=64),
    "fp32_ragged": small(dtype="f32", N=777, block_q=100, P=3),
    "bq1": small(N=50, block_q=1, P=2),
    "m0_512_bq256": small(M0=512, Ch=8, P=64, block_q=256, N=1536, d=128, B=1, H=2),
    "m0_300_bq128": small(M0=300, Ch=4, P=30, block_q=128, N=1024, B=1, H=2),
    # the largest ragged codebook the parent stream kernel holds (padding rows
    # in its last 32-row pair), and the smallest codebook
    "m0_500_d128": small(M0=500, Ch=8, P=40, block_q=128, N=1200, d=128, B=1, H=2),
    "m0_one": small(M0=1, Ch=2, P=1, N=300, B=1, H=2),
    # few heads: the aggregation splits the parents over several workgroups
    "m0_24_split": small(M0=24, Ch=2, P=5, B=1, H=1, N=700),
    "m0_44_split": small(M0=44, Ch=4, P=5, B=1, H=1, N=700),
    "fp32_ch16_d64": small(dtype="f32", M0=70, Ch=16, P=9, N=600),
    # fp32 at d = 128 stages one chunk at a time: several parent, importance
    # and child chunks
    "fp32_d128_multichunk": small(dtype="f32", d=128, M0=130, Ch=8, P=10, N=700, block_q=64),
    "fp32_d128_ch16_multichunk": small(dtype="f32", d=128, M0=70, Ch=16, P=9, N=500),
    "fp32_d128_bq256_multichunk": small(dtype="f32", d=128, M0=200, Ch=4, P=20, N=600,
                                        block_q=256),
    # an fp32 codebook past the stream kernel's LDS share: the one-shot parent
    # kernel (bf16 codebooks of every supported size stream)
    "fp32_m0_320_d64": small(dtype="f32", M0=320, Ch=2, P=24, N=900, B=1, H=2),
    # flat codebook (Ch = 0): VQ attention over the parents alone
    "flat": small(Ch=0, P=0),
    "flat_n_one": small(Ch=0, P=0, N=1, B=1, H=1),
    "flat_fp32_ragged": small(Ch=0, P=0, dtype="f32", N=777, block_q=100),
    "flat_fp32_d128": small(Ch=0, P=0, dtype="f32", d=128, block_q=64),
    "flat_m0_300_split": small(Ch=0, P=0, M0=300, B=1, H=1, N=2000),
    "flat_m0_512_d128": small(Ch=0, P=0, M0=512, d=128, N=1536, B=1, H=2, block_q=256),
    # few workgroups and at least 256 keys per parent: two or four half waves
    # share a family in the aggregation (on a 256-CU device: two for 64 heads
    # of 32 parents, four for fewer)
    "agg_split2": small(M0=32, Ch=4, P=4, N=8192, B=8, H=8, block_q=256),
    "agg_split4": small(M0=8, Ch=8, P=3, N=4200, B=1, H=2, block_q=256),
    "agg_split4_ragged_fp32_d128": small(dtype="f32", M0=20, Ch=2, P=4, N=11000, d=128, B=1,
                                         H=1, block_q=256),
    "agg_split4_flat": small(Ch=0, P=0, M0=16, N=9000, B=1, H=2, block_q=256),
    "agg_split4_ch16": small(M0=10, Ch=16, P=3, N=2600, B=1, H=2),
    # every key of a head in one workgroup's range, more than its key queue
    # holds: the queue is bucketed and summed in the middle of the scan
    "agg_queue_overflow": small(M0=8, Ch=8, P=3, N=20000, B=1, H=2, block_q=256),
    "agg_queue_overflow_d128": small(M0=8, Ch=8, P=3, N=20000, B=1, H=2, block_q=256,
                                     d=128),
    "agg_queue_overflow_flat": small(Ch=0, P=0, M0=4, N=30000, B=1, H=1, block_q=256),
}


@pytest.mark.parametrize("name", list(EDGE))
def test_edge_case(name):
    w = EDGE[name]
    banner(name, w)
    x = inputs.generate(w)
    res = parity.compare(x, w)
    report(res)


# the two-kernel precompute (avq_assign, then avq_aggregate) on cases that
# cover its paths; every other case runs the fused one
UNFUSED = ["ragged_n", "ch1", "ch2", "m0_37_ch16_d128", "fp32_d128", "m0_512_bq256",
           "agg_split4", "agg_queue_overflow", "flat", "dirichlet_sparse"]


@pytest.mark.parametrize("name", UNFUSED)
def test_edge_case_unfused(name):
    w = EDGE[name]
    banner(name + " (unfused)", w)
    res = parity.compare(inputs.generate(w), w, fused=False)
    report(res)


@pytest.mark.parametrize("name", ["ragged_n", "ch1", "ch2", "ch8_bq200", "m0_512_bq256",
                                  "agg_split2", "agg_split4", "agg_queue_overflow",
                                  "agg_queue_overflow_d128", "dirichlet_sparse", "keys_stay",
                                  "large_logits"])
def test_fused_equals_unfused(name):
    """avq_assign_aggregate gives avq_assign's indices and avq_aggregate's
    counts exactly (the same child compare routine on the same inputs), and
    the sums within fp32 summation-order rounding: each is a sum of the same
    values, so |a - b| <= 2 gamma_n sum |v| per element."""
    from paper_2607_12789_amd import avq
    w = EDGE[name]
    banner(name + " (fused vs unfused)", w)
    xd = parity.to_gpu(inputs.generate(w))
    p1, c1, pk1, n1, vb1 = avq.assign_aggregate(xd["K"], xd["V"], xd["Cp"], xd["Cc"], sums=True)
    p2, c2 = avq.assign(xd["K"], xd["Cp"], xd["Cc"])
    pk2, n2, vb2 = avq.aggregate(xd["V"], c2, w.M0, w.Ch, sums=True)
    torch.cuda.synchronize()
    assert torch.equal(p1, p2) and torch.equal(c1, c2) and torch.equal(n1, n2)
    # |v| summed per code with the GPU's codes (fp64 on the CPU)
    V = xd["V"].double().cpu()
    code = c1.long().cpu()
    Mtot = w.M0 * (1 + w.Ch)
    absum = torch.zeros((w.B, w.H, Mtot, w.d), dtype=torch.float64)
    absum.scatter_add_(2, code[..., None].expand(-1, -1, -1, w.d), V.abs())
    if w.Ch > 0:  # parent rows cover the whole cell
        par = torch.where(code < w.M0, code, (code - w.M0) // w.Ch)
        cell = torch.zeros_like(absum)
        cell.scatter_add_(2, par[..., None].expand(-1, -1, -1, w.d), V.abs())
        absum[:, :, :w.M0] = cell[:, :, :w.M0]
    bound = 2 * parity.gamma(w.N) * absum + 1e-30
    diff = (vb1.double().cpu() - vb2.double().cpu()).abs()
    assert (diff <= bound).all(), float((diff / bound).max())
    print(f"  indices, counts equal; Vbar max |diff|/bound = {float((diff / bound).max()):.3g}",
          flush=True)


def test_children_equal_parent_gives_vq_attention():
    """No key may move when the children equal their parent; the refined
    output then equals P = 0 VQ attention for every P."""
    w = small(Ch=8, P=6)
    banner("children_equal_parent", w)
    x = inputs.generate(w)
    x["Cc"] = x["Cp"][:, :, None, :].expand(-1, -1, w.Ch, -1).contiguous()
    res = parity.compare(x, w)
    report(res)
    g = res["gpu"]
    assert (g["code_idx"] < w.M0).all()
    assert (g["counts"][..., w.M0:] == 0).all()
    from paper_2607_12789_amd import avq
    xd = {k: v.cuda() for k, v in x.items()}
    packed = g["packed"].cuda()
    y_ref = avq.attention_fwd(xd["Q"], xd["Cp"], xd["Cc"], packed, w.P, w.block_q)
    y0 = avq.attention_fwd(xd["Q"], xd["Cp"], xd["Cc"], packed, 0, w.block_q)
    assert torch.equal(y_ref, y0)


@pytest.mark.parametrize("dtype,P,Ch", [("bf16", 16, 8), ("f32", 16, 8), ("bf16", 6, 8),
                                        ("bf16", 16, 4), ("f32", 6, 4), ("bf16", 9, 2),
                                        ("f32", 9, 2)])
def test_empty_far_children(dtype, P, Ch):
    """App. D: two children of a parent that the tiles select lie 100 units
    out on either side of it along the first axis, where every query has
    component +-3, so no key moves to them and one of them has a logit about
    300 natural units above every non-empty code's. The running max must skip
    empty children and their correcting weights must be exactly zero;
    otherwise the rescale underflows the accumulators and Y = 0/0."""
    import oracle
    w = small(dtype=dtype, M0=16, Ch=Ch, P=P, N=600, B=1, H=2)
    banner(f"empty_far_children_{dtype}_P{P}_Ch{Ch}", w)
    x = inputs.generate(w)
    Q = x["Q"].clone()
    sign = torch.where(torch.arange(w.N) % 2 == 0, 3.0, -3.0)
    Q[..., 0] = sign.to(Q.dtype)
    x = dict(x, Q=Q.contiguous())
    # the parent selected most often (importance does not depend on the children)
    o0 = oracle.forward(x["Q"], x["K"], x["V"], x["Cp"], x["Cc"], w.P, w.block_q)
    p = int(np.bincount(o0["selection"].reshape(-1), minlength=w.M0).argmax())
    Cc = x["Cc"].clone()
    far = torch.zeros(w.d, dtype=Cc.dtype)
    far[0] = 100.0
    Cc[:, p, 0] = x["Cp"][:, p] + far
    Cc[:, p, 1] = x["Cp"][:, p] - far
    x = dict(x, Cc=Cc.contiguous())
    res = parity.compare(x, w)
    report(res)
    o = res["oracle"]
    first = w.M0 + p * w.Ch
    assert (o["counts"][:, :, first:first + 2] == 0).all()  # both far children are empty
    assert (o["selection"] == p).any(axis=-1).sum() >= 2, "the far children's parent is not selected"


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_exact_ties_resolve_to_lowest_index(dtype):
    """Dyadic inputs, exact in every precision: exact distance ties and
    duplicate codewords must resolve exactly as the oracle does."""
    w = small(dtype=dtype, M0=12, Ch=4, P=3, N=900)
    banner(f"exact_ties_{dtype}", w)
    x = inputs.dyadic_exact(w.B, w.H, w.N, w.d, w.M0, w.Ch, seed=5, dtype=dtype)
    Cp = x["Cp"].clone()
    Cp[:, 7] = Cp[:, 2]  # duplicate parent
    x["Cp"] = Cp
    Cc = x["Cc"].clone()
    Cc[:, 4, 3] = Cc[:, 4, 1]  # duplicate child
    x["Cc"] = Cc
    res = parity.compare(x, w)
    report(res)
    assert res["assign"]["differing"] == 0
    g = res["gpu"]
    assert not (g["parent_idx"] == 7).any()


def test_repeat_runs_identical_integers():
    w = small(Ch=8, P=6)
    x = {k: v.cuda() for k, v in inputs.generate(w).items()}
    a = parity.gpu_forward(x, w)
    b = parity.gpu_forward(x, w)
    for k in ("parent_idx", "code_idx", "counts", "topp"):
        assert torch.equal(a[k], b[k]), k
    torch.testing.assert_close(a["Y"], b["Y"], rtol=2e-3, atol=1e-5)


# App. B importance (tiles of 64 parents) against the oracle's tiled importance
TILED = {
    "tiled_m0_256_d128": small(M0=256, Ch=8, P=32, d=128, N=2048, B=1, H=2),
    "tiled_m0_300_ragged": small(M0=300, Ch=4, P=30, N=1024, B=1, H=2),
    "tiled_fp32_d64": small(dtype="f32", M0=150, Ch=4, P=12, N=900),
    "tiled_p0_importance": small(M0=200, P=0, N=700),
    "tiled_bq200": small(M0=130, Ch=8, P=11, block_q=200, N=1300),
    "tiled_m0_512_bq256": small(M0=512, Ch=8, P=64, block_q=256, N=1536, d=128, B=1, H=2),
    "tiled_fp32_d128_ragged": small(dtype="f32", d=128, M0=130, Ch=8, P=10, N=700,
                                    block_q=64),
    "tiled_fp32_d128_bq256": small(dtype="f32", d=128, M0=200, Ch=4, P=20, N=600, block_q=256),
}


@pytest.mark.parametrize("name", list(TILED))
def test_tiled_importance(name):
    w = TILED[name]
    banner(name, w)
    x = inputs.generate(w)
    res = parity.compare(x, w, tiled=True)
    report(res)


def test_tiled_importance_empty_first_tile():
    """No key reaches the first 64 parents: their tile has N_seen = 0 and adds
    nothing; the later tiles extrapolate from the keys they have seen."""
    w = small(M0=200, Ch=4, P=20, N=900, B=1, H=2)
    banner("tiled_empty_first_tile", w)
    x = inputs.generate(w)
    Cp = x["Cp"].clone()
    Cp[:, :64] += 40.0
    x["Cp"] = Cp
    res = parity.compare(x, w, tiled=True)
    report(res)
    assert (res["oracle"]["counts"][..., :64] == 0).all()
    assert (res["gpu"]["importance"][..., :64] == 0).all()


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_tiled_single_tile_equals_exact(dtype):
    """M0 <= 64: one codeword tile, N_seen = N, and the two entry points give
    identical results."""
    from paper_2607_12789_amd import avq
    w = small(M0=64, Ch=8, P=6, dtype=dtype)
    xd = parity.to_gpu(inputs.generate(w))
    _, code = avq.assign(xd["K"], xd["Cp"], xd["Cc"])
    packed, _, _ = avq.aggregate(xd["V"], code, w.M0, w.Ch)
    a = avq.attention_fwd(xd["Q"], xd["Cp"], xd["Cc"], packed, w.P, w.block_q, debug=True)
    b = avq.attention_fwd(xd["Q"], xd["Cp"], xd["Cc"], packed, w.P, w.block_q, debug=True,
                          tiled_importance=True)
    for u, v in zip(a, b):
        assert torch.equal(u, v)


# Queries in a given order (Gilbert curve, or a random permutation) on
# spatially structured tokens: against the oracle run on the permuted queries
ORDERED = {
    "gilbert_64x64": (small(M0=64, Ch=8, P=16, N=4096, B=1, H=2, block_q=64, q_scale=8.0), 64, 64,
                      "gilbert", False),
    "gilbert_28x28_tiled": (small(M0=128, Ch=8, P=16, N=784, B=2, H=2, block_q=128,
                                  q_scale=8.0), 28, 28, "gilbert", True),
    "random_40x25_fp32": (small(dtype="f32", M0=96, Ch=4, P=12, N=1000, B=1, H=3, block_q=100,
                                q_scale=8.0), 40, 25, "random", False),
    "gilbert_32x32_flat": (small(Ch=0, P=0, M0=64, N=1024, B=1, H=2, block_q=64, q_scale=8.0),
                           32, 32, "gilbert", False),
}


@pytest.mark.parametrize("name", list(ORDERED))
def test_ordered_queries(name):
    from paper_2607_12789_amd import avq
    w, width, height, kind, tiled = ORDERED[name]
    banner(name, w)
    x = inputs.spatial(w, width, height)
    if kind == "gilbert":
        order = avq.gilbert_order(width, height)[0].numpy()
    else:
        order = np.random.default_rng(7).permutation(w.N).astype(np.int32)
    res = parity.compare(x, w, tiled=tiled, query_order=order)
    report(res)


def test_identity_order_equals_unordered():
    """query_order = 0 .. N-1 gives the unordered result bit for bit."""
    from paper_2607_12789_amd import avq
    w = small(Ch=8, P=6, N=700)
    xd = parity.to_gpu(inputs.generate(w))
    _, code = avq.assign(xd["K"], xd["Cp"], xd["Cc"])
    packed, _, _ = avq.aggregate(xd["V"], code, w.M0, w.Ch)
    ident = torch.arange(w.N, dtype=torch.int32, device="cuda")
    for tiled in (False, True):
        a = avq.attention_fwd(xd["Q"], xd["Cp"], xd["Cc"], packed, w.P, w.block_q, debug=True,
                              tiled_importance=tiled)
        b = avq.attention_fwd(xd["Q"], xd["Cp"], xd["Cc"], packed, w.P, w.block_q, debug=True,
                              tiled_importance=tiled, query_order=ident)
        for u, v in zip(a, b):
            assert torch.equal(u, v)


def test_order_entries_out_of_range_are_skipped():
    """An entry outside [0, N) takes no part: its query position writes no
    row; every other token's row equals the one of the valid permutation."""
    from paper_2607_12789_amd import avq
    w = small(Ch=4, P=0, N=500, B=1, H=1)
    xd = parity.to_gpu(inputs.generate(w))
    _, code = avq.assign(xd["K"], xd["Cp"], xd["Cc"])
    packed, _, _ = avq.aggregate(xd["V"], code, w.M0, w.Ch)
    ident = torch.arange(w.N, dtype=torch.int32, device="cuda")
    bad = ident.clone()
    bad[17] = w.N + 5
    bad[300] = -3
    y0 = avq.attention_fwd(xd["Q"], xd["Cp"], xd["Cc"], packed, 0, w.block_q, query_order=ident)
    y1 = torch.full_like(y0, 7.0)
    avq.attention_fwd(xd["Q"], xd["Cp"], xd["Cc"], packed, 0, w.block_q, Y=y1, query_order=bad)
    keep = torch.ones(w.N, dtype=torch.bool)
    keep[[17, 300]] = False
    assert torch.equal(y1[:, :, keep.cuda()], y0[:, :, keep.cuda()])
    assert (y1[:, :, 17] == 7.0).all() and (y1[:, :, 300] == 7.0).all()


# The five evaluation workloads run last (largest oracle work): every tile.
@pytest.mark.parametrize("name", ["c1", "c2", "c3", "c4", "c5"])
def test_workload(name):
    w = inputs.WORKLOADS[name]
    banner(name, w)
    x = inputs.generate(w)
    res = parity.compare(x, w)
    report(res)
    assert res["output"]["rows"] == w.B * w.H * w.N
    assert res["topp"]["tiles"] == w.B * w.H * w.n_tiles


@pytest.mark.parametrize("Ch", [0, 4])
def test_aggregate_ignores_out_of_range_codes(Ch):
    """Codes outside [0, Mtot) (here -1, -7, Mtot, 2^30) take no part: counts
    and sums equal those of the valid codes alone (numpy add.at reference)."""
    from paper_2607_12789_amd import avq
    from tests import references as ref
    w = small(Ch=Ch, P=0, M0=24, N=900, B=1, H=2, dtype="f32")
    x = inputs.generate(w)
    rng = np.random.default_rng(3)
    code = rng.integers(0, w.Mtot, size=(w.B, w.H, w.N)).astype(np.int32)
    bad = rng.random((w.B, w.H, w.N)) < 0.1
    code[bad] = rng.choice(np.array([-1, -7, w.Mtot, 1 << 30], np.int32), size=int(bad.sum()))
    V = x["V"].cuda()
    _, counts, Vbar = avq.aggregate(V, torch.from_numpy(code).cuda(), w.M0, w.Ch, sums=True)
    torch.cuda.synchronize()
    good = ~bad
    par = np.where(code < w.M0, code, (code - w.M0) // max(w.Ch, 1)).astype(np.int64)
    Vn = x["V"].double().numpy()
    exp_V, exp_n = np.zeros((w.B, w.H, w.Mtot, w.d)), np.zeros((w.B, w.H, w.Mtot), np.int64)
    for b in range(w.B):
        for h in range(w.H):
            g = good[b, h]
            rv, rn = ref.aggregates(Vn[b:b + 1, h:h + 1][:, :, g], par[b:b + 1, h:h + 1][:, :, g],
                                    code[b:b + 1, h:h + 1][:, :, g].astype(np.int64), w.M0, w.Ch)
            exp_V[b, h], exp_n[b, h] = rv[0, 0], rn[0, 0]
    np.testing.assert_array_equal(counts.cpu().numpy(), exp_n)
    np.testing.assert_allclose(Vbar.cpu().numpy(), exp_V, rtol=1e-5, atol=1e-4)


@pytest.mark.parametrize("dtype,Ch,d", [("bf16", 8, 128), ("f32", 4, 64), ("bf16", 0, 64),
                                        ("bf16", 16, 64), ("f32", 2, 128)])
def test_pack_aggregates_path(dtype, Ch, d):
    """Alg. 2 takes the aggregates as (Vbar, n): avq_aggregate's fp32 sums and
    counts packed by avq_pack_aggregates give exactly the bytes of its own
    packed output, and the attention from them is bit-equal and passes parity
    against the oracle."""
    import oracle
    from paper_2607_12789_amd import avq
    w = small(dtype=dtype, Ch=Ch, d=d, P=0 if Ch == 0 else 5, M0=40)
    banner(f"pack_aggregates_{dtype}_ch{Ch}_d{d}", w)
    x = inputs.generate(w)
    xd = parity.to_gpu(x)
    par, code = avq.assign(xd["K"], xd["Cp"], xd["Cc"])
    packed, counts, Vbar = avq.aggregate(xd["V"], code, w.M0, w.Ch, sums=True)
    packed2 = avq.pack_aggregates(Vbar, counts, w.M0, w.Ch, w.torch_dtype)
    torch.cuda.synchronize()
    assert torch.equal(packed, packed2)
    y1, t1, i1 = avq.attention_fwd(xd["Q"], xd["Cp"], xd["Cc"], packed, w.P, w.block_q, debug=True)
    y2, t2, i2 = avq.attention_fwd(xd["Q"], xd["Cp"], xd["Cc"], packed2, w.P, w.block_q,
                                   debug=True)
    assert torch.equal(y1, y2) and torch.equal(t1, t2) and torch.equal(i1, i2)
    # the packed path's own output against the oracle on the same codes and
    # selection (the certification of both is the general parity test's)
    res = parity.compare(x, w)
    report(res)
    g = dict(parent_idx=par.cpu(), code_idx=code.cpu(), topp=t2.cpu(), Y=y2.cpu())
    mask = np.ones((w.B, w.H, w.n_tiles), np.uint8)
    o = parity.oracle_on_gpu_codes(x, w, g, mask, True, None)
    sel = g["topp"].numpy() if w.P > 0 else o["selection"]
    oY, _ = oracle.output(x["Q"], x["Cp"], x["Cc"], o["Vbar"], o["counts"], sel, w.block_q)
    ry = parity.check_output(x, w, g, dict(o, Y=oY), mask.astype(bool))
    print(f"  pack path output: {ry.line()}", flush=True)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_pack_aggregates_caller_values(dtype):
    """Aggregates from the caller (random sums, counts with zeros and negative
    entries): every mean is fl(fl(Vbar) * fl(1/n)) rounded to the storage type
    (numpy fp32 arithmetic, then torch's round to nearest even), n exact,
    ln n within a few ulp, empty codes and padding 0 and -inf."""
    from paper_2607_12789_amd import avq
    B, H, M0, Ch, d = 2, 3, 37, 4, 64
    Mtot = M0 * (1 + Ch)
    rng = np.random.default_rng(11)
    Vbar = (rng.standard_normal((B, H, Mtot, d)) * 50).astype(np.float32)
    counts = rng.integers(-3, 300, size=(B, H, Mtot)).astype(np.int32)
    counts[rng.random((B, H, Mtot)) < 0.2] = 0
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    pk = avq.pack_aggregates(torch.from_numpy(Vbar).cuda(), torch.from_numpy(counts).cuda(), M0,
                             Ch, tdt)
    torch.cuda.synchronize()
    means, n_pk, ln_pk, pad = parity.unpack_packed(pk.cpu().numpy(), M0, Ch, d, dtype)
    n = np.maximum(counts, 0)
    inv = np.where(n > 0, np.float32(1) / np.maximum(n, 1).astype(np.float32), np.float32(0))
    m32 = (Vbar * inv[..., None].astype(np.float32)).astype(np.float32)
    expect = torch.from_numpy(m32).to(tdt).double().numpy()
    np.testing.assert_array_equal(means, expect)
    np.testing.assert_array_equal(n_pk, n.astype(np.float32))
    nz = n > 0
    assert np.isneginf(ln_pk[~nz]).all()
    err = np.abs(ln_pk[nz].astype(np.float64) - np.log(n[nz]))
    assert (err <= 8 * 2.0 ** -24 * np.maximum(np.log(n[nz]), 1)).all()
    assert (pad["means"] == 0).all() and (pad["n"] == 0).all() and np.isneginf(pad["ln"]).all()
