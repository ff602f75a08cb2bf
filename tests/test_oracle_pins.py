"""Pins of the fp64 oracle against what the paper and the mathematics fix.

Each check goes through a route other than the oracle's own formulas (library
routines, exhaustive enumeration, closed forms, invariants), so that a dropped
term, a wrong sign or index, or a transposed operand in the oracle fails at
least one of them. ``test_oracle_mutants.py`` plants such mistakes in copies
of the oracle and checks that these pins catch them.
"""
import itertools

import numpy as np
import pytest
import torch

import oracle
from paper_2607_12789_amd import inputs
from tests import references as ref


def small(**kw):
    base = dict(name="pin", B=1, H=2, N=100, d=8, M0=6, Ch=4, P=2, block_q=32,
                dtype="f32", sigma_c=0.3, sigma_k=0.2, q_scale=2.0, seed=3)
    base.update(kw)
    return inputs.Workload(**base)


def np64(t):
    return oracle.f64(t)


def run(x, w, recovered=True):
    return oracle.forward(x["Q"], x["K"], x["V"], x["Cp"], x["Cc"], w.P, w.block_q,
                          recovered=recovered)


# ---------------------------------------------------------------- assignment

@pytest.mark.parametrize("seed", [0, 1, 2])
def test_assign_matches_cdist(seed):
    """Sec. 3.2 assignment and Alg. 1 tree refinement against scipy cdist."""
    w = small(seed=seed)
    x = inputs.generate(w)
    o = oracle.assign(x["K"], x["Cp"], x["Cc"])
    par, code = ref.tree_assign(np64(x["K"]), np64(x["Cp"]), np64(x["Cc"]))
    np.testing.assert_array_equal(o["parent_idx"], par)
    np.testing.assert_array_equal(o["code_idx"], code)
    assert (code >= w.M0).any() and (code < w.M0).any()  # both branches exercised


def test_assign_exact_ties_lowest_index():
    """Dyadic inputs: exact ties between codewords resolve to the lowest index,
    and equal child/parent distances keep the key on its parent (strict <)."""
    x = inputs.dyadic_exact(B=1, H=2, N=300, d=4, M0=5, Ch=4, seed=7)
    Cp = x["Cp"].clone()
    Cp[0, 3] = Cp[0, 1]  # duplicate parent: index 3 can never win
    x["Cp"] = Cp
    o = oracle.assign(x["K"], x["Cp"], x["Cc"])
    par, code = ref.tree_assign(np64(x["K"]), np64(x["Cp"]), np64(x["Cc"]))
    np.testing.assert_array_equal(o["parent_idx"], par)
    np.testing.assert_array_equal(o["code_idx"], code)
    assert not (o["parent_idx"][0, 0] == 3).any()
    # some exact parent ties and some exact child/parent ties actually occur
    ties = o["d_parent2"] == o["d_parent"]
    assert ties.any()
    stay_tie = (o["d_child"] == o["d_parent"])
    assert stay_tie.any()
    assert (o["code_idx"][stay_tie] < 5).all()


def test_assign_codebook_equals_keys():
    """Codebook made of the keys themselves: every key is its own codeword."""
    rng = np.random.default_rng(0)
    K = rng.standard_normal((1, 1, 40, 6))
    Cp = K[0].copy()
    Cc = np.repeat(Cp[:, :, None, :], 2, axis=2)
    o = oracle.assign(K, Cp, Cc)
    np.testing.assert_array_equal(o["parent_idx"][0, 0], np.arange(40))
    np.testing.assert_array_equal(o["code_idx"][0, 0], np.arange(40))
    assert (o["d_parent"] == 0).all()


# ---------------------------------------------------------------- aggregates

def test_aggregates_match_add_at_and_invariants():
    """Eq. (aggregates): bincount/add.at route; sum of parent counts is N per
    head; parent rows sum to the total value; children never exceed parents."""
    w = small(B=2, H=3, N=257, sigma_k=0.2)
    x = inputs.generate(w)
    o = oracle.assign(x["K"], x["Cp"], x["Cc"])
    Vbar, n = oracle.aggregate(x["V"], o["parent_idx"], o["code_idx"], w.M0, w.Ch)
    Vr, nr = ref.aggregates(np64(x["V"]), o["parent_idx"].astype(np.int64),
                            o["code_idx"].astype(np.int64), w.M0, w.Ch)
    np.testing.assert_array_equal(n, nr)
    np.testing.assert_allclose(Vbar, Vr, rtol=0, atol=1e-12)
    assert (n[..., :w.M0].sum(-1) == w.N).all()
    np.testing.assert_allclose(Vbar[..., :w.M0, :].sum(-2), np64(x["V"]).sum(-2), atol=1e-10)
    child = n[..., w.M0:].reshape(w.B, w.H, w.M0, w.Ch).sum(-1)
    assert (child <= n[..., :w.M0]).all()


# ---------------------------------------------------------------- importance

@pytest.mark.parametrize("block_q", [32, 100, 7])
def test_importance_equals_per_key_attention_mass(block_q):
    """Eq. (importance) equals the softmax mass that a tile's queries put on
    the keys of each parent cell (per-key route through torch.softmax), and it
    sums to the tile size (attention weights sum to 1)."""
    w = small(block_q=block_q)
    x = inputs.generate(w)
    o = run(x, w)
    Q, Cp = np64(x["Q"]), np64(x["Cp"])
    T = w.n_tiles
    for b in range(w.B):
        for h in range(w.H):
            for t in range(T):
                rows = slice(t * block_q, min((t + 1) * block_q, w.N))
                wr = ref.per_key_importance(Q[b, h, rows], Cp[h], o["parent_idx"][b, h])
                np.testing.assert_allclose(o["importance"][b, h, t], wr, rtol=1e-10,
                                           atol=1e-13)
                n_rows = rows.stop - rows.start
                assert abs(o["importance"][b, h, t].sum() - n_rows) < 1e-9 * n_rows


def test_importance_zero_for_empty_parents():
    w = small(M0=12, N=40)
    x = inputs.generate(w)
    o = run(x, w)
    empty = o["counts"][..., :w.M0] == 0
    assert empty.any()
    wimp = o["importance"]
    for t in range(w.n_tiles):
        assert (wimp[:, :, t][empty] == 0).all()


def _tiled_inputs(**kw):
    w = small(M0=10, N=150, block_q=40, **kw)
    x = inputs.generate(w)
    o = run(x, w)
    return w, x, o, o["counts"]


@pytest.mark.parametrize("tile_c", [10, 16])
def test_tiled_importance_single_tile_is_exact(tile_c):
    """App. B: with every parent in one tile, N_seen = N after it and the
    extrapolated denominator is the exact one: Eq. (importance)."""
    w, x, o, n = _tiled_inputs()
    wt = oracle.importance_tiled(x["Q"], x["Cp"], n, w.Ch, w.block_q, tile_c)
    np.testing.assert_allclose(wt, o["importance"], rtol=1e-12, atol=1e-15)


@pytest.mark.parametrize("tile_c", [1, 3, 4])
def test_tiled_importance_last_tile_is_exact(tile_c):
    """The tile processed last has seen every key (N_seen = N): its parents
    get their Eq. (importance) values; earlier tiles differ in general."""
    w, x, o, n = _tiled_inputs()
    wt = oracle.importance_tiled(x["Q"], x["Cp"], n, w.Ch, w.block_q, tile_c)
    last = ((w.M0 - 1) // tile_c) * tile_c
    np.testing.assert_allclose(wt[..., last:], o["importance"][..., last:], rtol=1e-12,
                               atol=1e-15)
    assert not np.allclose(wt[..., :last], o["importance"][..., :last], rtol=1e-6)


def test_tiled_importance_first_tile_closed_form():
    """tile_c = 1: after the first parent, Ztilde_i = N/n_0 * n_0 e^S_i0, so
    w_0 = |I| n_0 / N whatever the logits; a tile of empty parents gets 0."""
    w, x, o, n = _tiled_inputs(seed=4)
    wt = oracle.importance_tiled(x["Q"], x["Cp"], n, w.Ch, w.block_q, 1)
    sizes = np.array([min(w.block_q, w.N - t * w.block_q) for t in range(w.n_tiles)])
    for b in range(w.B):
        for h in range(w.H):
            first = int(np.argmax(n[b, h, :w.M0] > 0))
            expect = sizes * n[b, h, first] / w.N
            np.testing.assert_allclose(wt[b, h, :, first], expect, rtol=1e-12)
            assert (wt[b, h, :, :w.M0][:, n[b, h, :w.M0] == 0] == 0).all()


@pytest.mark.parametrize("tile_c", [1, 3])
def test_tiled_importance_zero_queries(tile_c):
    """Q = 0: every logit is 0, each partial denominator is exactly N_seen,
    Ztilde = N, and tiled importance equals exact importance = |I| n_a / N."""
    w, x, o, n = _tiled_inputs()
    Q0 = torch.zeros_like(x["Q"])
    wt = oracle.importance_tiled(Q0, x["Cp"], n, w.Ch, w.block_q, tile_c)
    we = oracle.importance(Q0, x["Cp"], n, w.Ch, w.block_q)
    np.testing.assert_allclose(wt, we, rtol=1e-12, atol=1e-15)
    sizes = np.array([min(w.block_q, w.N - t * w.block_q) for t in range(w.n_tiles)])
    np.testing.assert_allclose(wt, sizes[None, None, :, None] * n[:, :, None, :w.M0] / w.N,
                               rtol=1e-12)


def test_capture_of_full_selection_is_one():
    """Capture (App. B): selecting every parent captures all attention mass;
    the best selection of P parents captures at least as much as any other."""
    w, x, o, n = _tiled_inputs()
    T = w.n_tiles
    full = np.broadcast_to(np.arange(w.M0, dtype=np.int32), (w.B, w.H, T, w.M0))
    cap = oracle.capture(x["Q"], x["K"], o["parent_idx"], full, w.block_q)
    assert abs(cap["selected"] - 1.0) < 1e-12 and abs(cap["exact"] - 1.0) < 1e-12
    sel = oracle.topp(o["importance"], 3)
    cap3 = oracle.capture(x["Q"], x["K"], o["parent_idx"], sel, w.block_q)
    assert 0 < cap3["selected"] <= cap3["exact"] + 1e-12 < 1


# ---------------------------------------------------------------- top-P

def _capture_by_subsets(Q, K, par, M0, P, block_q):
    """Best capture by exhaustive search: per tile, the attention mass each
    query puts on each parent cell comes from SDPA with one-hot parent values
    (softmax over the original keys, Eq. (standardattention)); every P-subset
    of parents is tried and the largest total mass over the tile kept."""
    N = Q.shape[0]
    onehot = np.eye(M0)[par]
    total, count = 0.0, 0
    for t0 in range(0, N, block_q):
        mass = ref.sdpa(Q[t0:t0 + block_q], K, onehot)  # [queries, M0]
        best = max(mass[:, list(sub)].sum() for sub in itertools.combinations(range(M0), P))
        total += best
        count += mass.shape[0]
    return total / count


@pytest.mark.parametrize("P", [1, 2, 4])
def test_capture_best_selection_by_enumeration(P):
    """Capture (App. B, tab. tiled_capture): the "exact" figure is the best
    P-subset of parents per tile, found by trying every subset; a selection
    given to it is scored by the same SDPA masses."""
    w = small(N=70, M0=7, Ch=2, P=P, block_q=16, d=6, q_scale=4.0)
    x = inputs.generate(w)
    o = run(x, w)
    sel = np.broadcast_to(np.arange(P, dtype=np.int32)[::-1], (w.B, w.H, w.n_tiles, P))
    cap = oracle.capture(x["Q"], x["K"], o["parent_idx"], sel, w.block_q)
    Q, K = np64(x["Q"]), np64(x["K"])
    exact, got, count = 0.0, 0.0, 0
    for h in range(w.H):
        exact += _capture_by_subsets(Q[0, h], K[0, h], o["parent_idx"][0, h], w.M0, P,
                                     w.block_q) * w.N
        onehot = np.eye(w.M0)[o["parent_idx"][0, h]]
        got += ref.sdpa(Q[0, h], K[0, h], onehot)[:, :P].sum()
        count += w.N
    np.testing.assert_allclose(cap["exact"], exact / count, rtol=1e-12)
    np.testing.assert_allclose(cap["selected"], got / count, rtol=1e-12)
    assert cap["selected"] < cap["exact"]  # the fixed selection is not the best here


def test_capture_hand_worked():
    """Two queries, three keys in two parent cells, logits chosen so that the
    masses are simple fractions:
      query 0: logits (ln 1, ln 1, ln 8) on keys (cell 0, cell 0, cell 1)
               -> masses cell 0: 2/10, cell 1: 8/10;
      query 1: logits (ln 3, ln 3, ln 4) -> cell 0: 6/10, cell 1: 4/10.
    Tile sums: cell 0: 0.8, cell 1: 1.2, so with P = 1 the best selection of
    the tile is cell 1 (capture (0.8 + 0.4) / 2 = 0.6), although it holds fewer
    keys and query 1 alone prefers cell 0 (each query's own best would give
    0.7). Selecting cell 0 captures (0.2 + 0.6) / 2 = 0.4."""
    K = np.array([[1.0, 0.0], [1.0, 0.0], [0.0, 1.0]])
    Q = np.array([[0.0, np.log(8.0)], [np.log(3.0), np.log(4.0)]])
    par = np.array([0, 0, 1], np.int32)[None, None]
    Qb, Kb = Q[None, None], K[None, None]
    c1 = oracle.capture(Qb, Kb, par, np.array([[[[1]]]], np.int32), block_q=2)
    c0 = oracle.capture(Qb, Kb, par, np.array([[[[0]]]], np.int32), block_q=2)
    assert abs(c1["exact"] - 0.6) < 1e-12 and abs(c0["exact"] - 0.6) < 1e-12
    assert abs(c1["selected"] - 0.6) < 1e-12
    assert abs(c0["selected"] - 0.4) < 1e-12


@pytest.mark.parametrize("P", [0, 1, 3, 6])
def test_topp_matches_enumeration(P):
    rng = np.random.default_rng(P)
    for trial in range(20):
        wv = rng.random(6)
        if trial % 3 == 0:
            wv = np.round(wv * 3) / 3  # exact ties
        if trial % 4 == 1:
            wv[rng.integers(0, 6, 2)] = 0.0
        sel = oracle.topp(wv[None], P)[0]
        np.testing.assert_array_equal(sel, ref.topp_by_enumeration(wv, P))


# ---------------------------------------------------------------- output

def test_p0_is_vq_attention():
    """P = 0: plain VQ attention of Sec. 3.2, i.e. per-key softmax attention
    with each key replaced by its parent codeword (SDPA route)."""
    w = small(P=0)
    x = inputs.generate(w)
    o = run(x, w)
    Q, V, Cp = np64(x["Q"]), np64(x["V"]), np64(x["Cp"])
    for b in range(w.B):
        for h in range(w.H):
            khat = Cp[h][o["parent_idx"][b, h]]
            np.testing.assert_allclose(o["Y"][b, h], ref.sdpa(Q[b, h], khat, V[b, h]),
                                       rtol=1e-10, atol=1e-12)


def test_flat_codebook_is_vq_attention():
    """Ch = 0 (a flat codebook, the VQ attention of Sec. 3.2): every key takes
    its nearest parent (scipy cdist), the aggregates are a bincount, and the
    output is per-key softmax attention with each key replaced by that
    codeword (SDPA route). It also equals the P = 0 output of the same keys
    and parents under a tree codebook, whose children P = 0 never reads."""
    w = small(Ch=0, P=0, N=130, block_q=32)
    x = inputs.generate(w)
    assert x["Cc"].shape == (w.H, w.M0, 0, w.d)
    o = run(x, w)
    Q, K, V, Cp = np64(x["Q"]), np64(x["K"]), np64(x["V"]), np64(x["Cp"])
    for b in range(w.B):
        for h in range(w.H):
            idx, _ = ref.nearest(K[b, h], Cp[h])
            np.testing.assert_array_equal(o["parent_idx"][b, h], idx)
            np.testing.assert_array_equal(o["code_idx"][b, h], idx)
            np.testing.assert_array_equal(o["counts"][b, h], np.bincount(idx, minlength=w.M0))
            np.testing.assert_allclose(o["Y"][b, h], ref.sdpa(Q[b, h], Cp[h][idx], V[b, h]),
                                       rtol=1e-10, atol=1e-12)
    tree = dict(x, Cc=x["Cp"][:, :, None, :].repeat(1, 1, 3, 1) * 1.5)
    ot = oracle.forward(tree["Q"], tree["K"], tree["V"], tree["Cp"], tree["Cc"], 0, w.block_q)
    np.testing.assert_allclose(o["Y"], ot["Y"], rtol=1e-12, atol=1e-14)
    assert o["selection"].shape[-1] == 0


def test_one_codeword_per_key_is_exact_attention():
    """Codebook = the keys (M0 = N, distinct keys) and P = 0: exact softmax
    attention, Eq. (standardattention), through torch SDPA."""
    rng = np.random.default_rng(5)
    N, d = 48, 8
    Q = rng.standard_normal((1, 1, N, d)) * 0.7
    K = rng.standard_normal((1, 1, N, d))
    V = rng.standard_normal((1, 1, N, d))
    Cp = K[0].copy()
    Cc = np.repeat(Cp[:, :, None, :], 2, axis=2)
    o = oracle.forward(Q, K, V, Cp, Cc, P=0, block_q=16)
    np.testing.assert_allclose(o["Y"][0, 0], ref.sdpa(Q[0, 0], K[0, 0], V[0, 0]),
                               rtol=1e-10, atol=1e-12)


@pytest.mark.parametrize("P", [1, 2, 6])
@pytest.mark.parametrize("block_q", [32, 13])
def test_refined_direct_equals_per_key_replacement(P, block_q):
    """App. C: updating with the correcting attention equals attention over
    keys where every key that moved to a child of a selected parent is
    represented by that child, and all others by their parent. Checked with the
    direct parent logit (App. C form) against SDPA per tile, using the oracle's
    own top-P sets, which the enumeration test pins."""
    w = small(P=P, block_q=block_q)
    x = inputs.generate(w)
    o = run(x, w, recovered=False)
    Q, V, Cp, Cc = np64(x["Q"]), np64(x["V"]), np64(x["Cp"]), np64(x["Cc"])
    for b in range(w.B):
        for h in range(w.H):
            for t in range(w.n_tiles):
                rows = slice(t * block_q, min((t + 1) * block_q, w.N))
                khat = ref.quantised_keys(Cp[h], Cc[h], o["parent_idx"][b, h],
                                          o["code_idx"][b, h], o["selection"][b, h, t])
                np.testing.assert_allclose(o["Y"][b, h, rows],
                                           ref.sdpa(Q[b, h, rows], khat, V[b, h]),
                                           rtol=1e-9, atol=1e-11)


def test_refined_recovered_per_key_weights():
    """Eq. (parent_recovery) form: per key, a moved key of a selected parent
    carries weight e^{T} + e^{S_p} - e^{mean_c T_c}; every other key e^{S_p}.
    Evaluated key by key in NumPy (no aggregates) and compared to the oracle."""
    w = small(P=2, block_q=20, sigma_c=0.5)
    x = inputs.generate(w)
    o = run(x, w, recovered=True)
    Q, V, Cp, Cc = np64(x["Q"]), np64(x["V"]), np64(x["Cp"]), np64(x["Cc"])
    for b in range(w.B):
        for h in range(w.H):
            par, code = o["parent_idx"][b, h], o["code_idx"][b, h]
            for t in range(w.n_tiles):
                sel = o["selection"][b, h, t]
                for i in range(t * w.block_q, min((t + 1) * w.block_q, w.N)):
                    q = Q[b, h, i]
                    sp = Cp[h][par] @ q
                    wgt = np.exp(sp)
                    for j in range(w.N):
                        if code[j] >= w.M0 and par[j] in sel:
                            c = code[j] - w.M0
                            tc = Cc[h, c // w.Ch, c % w.Ch] @ q
                            mean_t = (Cc[h, par[j]] @ q).mean()
                            wgt[j] = np.exp(tc) + np.exp(sp[j]) - np.exp(mean_t)
                    y = (wgt[:, None] * V[b, h]).sum(0) / wgt.sum()
                    np.testing.assert_allclose(o["Y"][b, h, i], y, rtol=1e-9, atol=1e-11)


def test_recovered_equals_direct_on_exact_constraint():
    """Eq. (parent_recovery) is exact when the parent is exactly the mean of its
    children: on dyadic codebooks the two forms agree to rounding."""
    x = inputs.dyadic_exact(B=1, H=2, N=200, d=8, M0=6, Ch=4, seed=11, dtype="f32")
    oa = oracle.forward(x["Q"], x["K"], x["V"], x["Cp"], x["Cc"], 3, 32, recovered=True)
    ob = oracle.forward(x["Q"], x["K"], x["V"], x["Cp"], x["Cc"], 3, 32, recovered=False)
    np.testing.assert_allclose(oa["Y"], ob["Y"], rtol=1e-13, atol=1e-13)
    assert (oa["code_idx"] >= 6).any()


def test_full_p_is_tree_vq_attention():
    """P = M0: every moved key is represented by its child, every other key by
    its parent, independent of importance (SDPA route)."""
    w = small(P=6)
    x = inputs.generate(w)
    o = run(x, w, recovered=False)
    Q, V, Cp, Cc = np64(x["Q"]), np64(x["V"]), np64(x["Cp"]), np64(x["Cc"])
    for b in range(w.B):
        for h in range(w.H):
            khat = ref.quantised_keys(Cp[h], Cc[h], o["parent_idx"][b, h], o["code_idx"][b, h])
            np.testing.assert_allclose(o["Y"][b, h], ref.sdpa(Q[b, h], khat, V[b, h]),
                                       rtol=1e-9, atol=1e-11)


def test_zero_queries_give_mean_value():
    """Q = 0: every logit is 0, so each key has weight 1 and Y is the plain mean
    of V for every P (parents count n, corrections vanish)."""
    w = small(P=3)
    x = inputs.generate(w)
    x["Q"] = torch.zeros_like(x["Q"])
    o = run(x, w)
    mean = np64(x["V"]).mean(axis=2, keepdims=True)
    np.testing.assert_allclose(o["Y"], np.broadcast_to(mean, o["Y"].shape), rtol=1e-12,
                               atol=1e-13)


def test_children_equal_parent_reduce_to_vq():
    """Children identical to their parent: no key moves (strict <), every child
    is empty, and the output equals P = 0 VQ attention for every P."""
    w = small(P=3)
    x = inputs.generate(w)
    x["Cc"] = x["Cp"][:, :, None, :].expand(-1, -1, w.Ch, -1).contiguous()
    o = run(x, w)
    assert (o["code_idx"] < w.M0).all()
    assert (o["counts"][..., w.M0:] == 0).all()
    o0 = oracle.forward(x["Q"], x["K"], x["V"], x["Cp"], x["Cc"], 0, w.block_q)
    np.testing.assert_allclose(o["Y"], o0["Y"], rtol=1e-13, atol=1e-14)


def test_linearity_in_values():
    w = small(P=2)
    x = inputs.generate(w)
    rng = np.random.default_rng(1)
    V2 = rng.standard_normal(x["V"].shape)
    o1 = run(x, w)
    x2 = dict(x, V=torch.from_numpy(V2))
    o2 = run(x2, w)
    x3 = dict(x, V=torch.from_numpy(2.0 * np64(x["V"]) - 3.0 * V2))
    o3 = run(x3, w)
    np.testing.assert_allclose(o3["Y"], 2.0 * o1["Y"] - 3.0 * o2["Y"], rtol=1e-10, atol=1e-11)
    x4 = dict(x, V=torch.full(x["V"].shape, 0.75, dtype=torch.float64))
    np.testing.assert_allclose(run(x4, w)["Y"], 0.75, rtol=1e-12)


def test_key_permutation_invariance_and_query_tile_equivariance():
    w = small(P=2, block_q=25)
    x = inputs.generate(w)
    o = run(x, w)
    rng = np.random.default_rng(2)
    perm = rng.permutation(w.N)
    xk = dict(x, K=x["K"][:, :, perm], V=x["V"][:, :, perm])
    np.testing.assert_allclose(run(xk, w)["Y"], o["Y"], rtol=1e-11, atol=1e-12)
    qperm = np.concatenate([t * 25 + rng.permutation(25) for t in range(4)])
    xq = dict(x, Q=x["Q"][:, :, qperm])
    np.testing.assert_allclose(run(xq, w)["Y"], o["Y"][:, :, qperm], rtol=1e-11, atol=1e-12)


def test_large_logits_stay_finite():
    """App. D: masked running max and zeroed empty codes keep Q x 20 finite."""
    w = small(P=3, M0=12, N=60)
    x = inputs.generate(w)
    x["Q"] = x["Q"] * 20
    o = run(x, w)
    assert np.isfinite(o["Y"]).all()
    assert (o["zratio"] > 0).all()


def test_empty_far_children_do_not_poison():
    """App. D: a selected parent whose children lie far away on both sides (so
    they are empty and the parent is still their exact mean) has child logits
    far above the running max. Their e^{T - m} overflows fp64; the empty-code
    mask must keep the output finite and equal to per-key attention."""
    rng = np.random.default_rng(4)
    d, M0, Ch, N = 4, 3, 2, 60
    Cp = rng.integers(-4, 5, size=(1, M0, d)).astype(np.float64)
    Cc = Cp[:, :, None, :] + np.array([0.25, -0.25])[None, None, :, None]
    far = np.zeros(d)
    far[0] = 512.0
    Cc[0, 0, 0] = Cp[0, 0] + far
    Cc[0, 0, 1] = Cp[0, 0] - far
    comp = rng.integers(0, M0, size=N)
    K = (Cp[0, comp] + rng.integers(-1, 2, size=(N, d)) / 8.0)[None, None]
    Q = np.zeros((1, 1, N, d))
    Q[0, 0, :, 0] = np.where(np.arange(N) % 2 == 0, 3.0, -3.0)
    Q[0, 0, :, 1:] = rng.integers(-2, 3, size=(N, d - 1)) / 4.0
    V = rng.standard_normal((1, 1, N, d))
    o = oracle.forward(Q, K, V, Cp, Cc, P=M0, block_q=16)
    assert o["counts"][0, 0, M0:M0 + Ch].sum() == 0  # both far children are empty
    assert np.isfinite(o["Y"]).all()
    for t in range(4):
        rows = slice(16 * t, min(16 * t + 16, N))
        khat = ref.quantised_keys(Cp[0], Cc[0], o["parent_idx"][0, 0], o["code_idx"][0, 0])
        np.testing.assert_allclose(o["Y"][0, 0, rows], ref.sdpa(Q[0, 0, rows], khat, V[0, 0]),
                                   rtol=1e-9, atol=1e-11)


# ---------------------------------------------------------------- codebook update

def _ema_state(H=2, M0=5, Ch=4, d=6, B=3, seed=0):
    """A random EMA state and batch statistics (positive masses)."""
    rng = np.random.default_rng(seed)
    Mtot = M0 * (1 + Ch)
    S = rng.standard_normal((H, Mtot, d)) * 3
    Nema = rng.uniform(0.5, 20.0, (H, Mtot))
    sums = rng.standard_normal((B, H, Mtot, d)) * 5
    counts = rng.integers(0, 30, (B, H, Mtot))
    return S, Nema, sums, counts


def test_codebook_update_keeps_the_constraint():
    """App. A: after the update every parent is the mean of its children."""
    S, Nema, sums, counts = _ema_state()
    _, _, Cp, Cc = oracle.codebook_update(sums, counts, S, Nema, 5, 4, 0.9)
    np.testing.assert_allclose(Cc.mean(axis=2), Cp, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("Ch", [1, 2, 4, 8])
def test_codebook_update_solves_the_weighted_least_squares(Ch):
    """Eq. (child_constraint_solve) is the minimiser of sum_c N_c ||M_c - C_c||^2
    under mean(C_c) = C_p: checked against the KKT system solved by
    numpy.linalg.solve, per parent and dimension."""
    M0, d = 3, 5
    S, Nema, sums, counts = _ema_state(M0=M0, Ch=Ch, d=d, seed=Ch)
    S2, N2, Cp, Cc = oracle.codebook_update(sums, counts, S, Nema, M0, Ch, 0.7)
    for h in range(S.shape[0]):
        for p in range(M0):
            rows = M0 + p * Ch + np.arange(Ch)
            Nc = N2[h, rows]
            M = S2[h, rows] / Nc[:, None]
            # unknowns C_1..C_Ch and the multiplier mu:
            # 2 N_c (C_c - M_c) + mu = 0;  sum_c C_c = Ch C_p
            A = np.zeros((Ch + 1, Ch + 1))
            A[:Ch, :Ch] = np.diag(2 * Nc)
            A[:Ch, Ch] = 1.0
            A[Ch, :Ch] = 1.0
            for e in range(d):
                rhs = np.concatenate([2 * Nc * M[:, e], [Ch * Cp[h, p, e]]])
                sol = np.linalg.solve(A, rhs)
                np.testing.assert_allclose(Cc[h, p, :, e], sol[:Ch], rtol=1e-10, atol=1e-10)


def test_codebook_update_ema_closed_form():
    """Constant inputs: S' = lambda S + (1 - lambda) B s and
    N' = lambda N + (1 - lambda) B n, worked by hand for lambda = 0.75,
    S = 4, N = 2, B = 3 batches of sums 8 and counts 5: S' = 9, N' = 5.25."""
    B, H, M0, Ch, d = 3, 1, 2, 2, 3
    Mtot = M0 * (1 + Ch)
    S = np.full((H, Mtot, d), 4.0)
    Nema = np.full((H, Mtot), 2.0)
    sums = np.full((B, H, Mtot, d), 8.0)
    counts = np.full((B, H, Mtot), 5)
    S2, N2, Cp, Cc = oracle.codebook_update(sums, counts, S, Nema, M0, Ch, 0.75)
    np.testing.assert_array_equal(S2, 9.0)
    np.testing.assert_array_equal(N2, 5.25)
    np.testing.assert_allclose(Cp, 9.0 / 5.25, rtol=1e-15)
    np.testing.assert_allclose(Cc, 9.0 / 5.25, rtol=1e-15)  # already constrained


def test_codebook_update_lambda_zero_gives_batch_means():
    """lambda = 0: the parents move to the mean of the keys of their cell and
    the children, whose cells hold keys, to a projection of their own means;
    compared with means computed from the keys by numpy grouping."""
    w = small(B=2, N=300, sigma_k=0.2)
    x = inputs.generate(w)
    a = oracle.assign(x["K"], x["Cp"], x["Cc"])
    sums, counts = oracle.aggregate(x["K"], a["parent_idx"], a["code_idx"], w.M0, w.Ch)
    Mtot = w.Mtot
    S0 = np.zeros((w.H, Mtot, w.d))
    N0 = np.ones((w.H, Mtot))
    _, N2, Cp, _ = oracle.codebook_update(sums, counts, S0, N0, w.M0, w.Ch, 0.0)
    K = np64(x["K"])
    for h in range(w.H):
        keys = K[:, h].reshape(-1, w.d)
        par = a["parent_idx"][:, h].reshape(-1)
        for p in range(w.M0):
            sel = par == p
            assert N2[h, p] == sel.sum()
            if sel.any():
                np.testing.assert_allclose(Cp[h, p], keys[sel].mean(axis=0), rtol=1e-12,
                                           atol=1e-12)


def test_codebook_update_equal_masses_shift_uniformly():
    """Equal child masses: the projection moves every child by the same
    amount, -delta / Ch (the plain Euclidean projection)."""
    S, Nema, sums, counts = _ema_state(M0=2, Ch=4)
    Nema[:] = 3.0
    counts[:] = 2
    S2, N2, Cp, Cc = oracle.codebook_update(sums, counts, S, Nema, 2, 4, 0.5)
    M = (S2[:, 2:] / N2[:, 2:, None]).reshape(2, 2, 4, -1)
    shift = Cc - M
    np.testing.assert_allclose(shift, np.broadcast_to(shift[:, :, :1], shift.shape), atol=1e-12)
    delta = M.sum(axis=2) - 4 * Cp
    np.testing.assert_allclose(shift[:, :, 0], -delta / 4, atol=1e-12)


def test_codebook_update_heavier_children_move_less():
    """Two children: each is displaced in inverse proportion to its mass."""
    S, Nema, sums, counts = _ema_state(M0=1, Ch=2, seed=3)
    S2, N2, Cp, Cc = oracle.codebook_update(sums, counts, S, Nema, 1, 2, 0.8)
    M = S2[:, 1:] / N2[:, 1:, None]
    d1 = np.linalg.norm(Cc[:, 0, 0] - M[:, 0], axis=-1)
    d2 = np.linalg.norm(Cc[:, 0, 1] - M[:, 1], axis=-1)
    np.testing.assert_allclose(d1 * N2[:, 1], d2 * N2[:, 2], rtol=1e-10)
