"""GPU-vs-oracle comparison helpers for the parity tests.

Decisions that floating point makes (nearest codeword, top-P membership) are
compared under a certification rule: a decision is *certified* when the
oracle's fp64 margin exceeds a bound on the kernel's fp32 rounding error, and
certified decisions must match bit for bit. An uncertified decision may go
either way; if the kernel's choice differs from the oracle's it must be a
valid choice within that bound, and everything downstream of it is then
compared with the oracle re-run on the kernel's choice: where codes differ,
the oracle's aggregates, importance, top-P and output are recomputed from the
GPU's codes (every head is compared); where a tile's top-P set differs, its
output rows are compared with the oracle's output for the GPU's selection
(every tile is compared). Nothing is left out. Integers are compared exactly,
floats within the stated tolerance.

Error bounds (u = 2^-24, gamma_n = n u / (1 - n u)):
* parent distances ||c||^2 - 2 k.c: products of bf16 inputs are exact in
  fp32 and the sums over d take gamma_d, so the error of one candidate is at
  most gamma_d (||c||^2 + 2 ||k|| ||c||) + u |value|;
* child and recomputed parent distances: fp32 sums of (k - c)^2 (error at
  most gamma_(d+1) times the distance) or, for bf16, ||c||^2 - 2 k.c from
  dot products of exact bf16 products (error at most
  (gamma_d + u)(||c||^2 + 2 ||k|| ||c||)); both bounds are added;
* importance: the logits carry gamma_d ||q|| ||c||, the weights exp(S - m)
  twice that plus the exp unit's rounding of (S - m) log2 e, and the
  normalised sums gamma_(M0 + block_q); w is compared relative to
  eps_w = 4 gamma_d max||q|| max||c|| + 2 u (max(m - S) + 8) + 2 gamma_(M0 + block_q).
"""
from __future__ import annotations

import math

import numpy as np
import torch

import oracle
from paper_2607_12789_amd import avq

U = 2.0 ** -24
TOL_Y = {"f32": 1e-4, "bf16": 2e-2}


def gamma(n):
    return n * U / (1 - n * U)


def to_gpu(x: dict) -> dict:
    return {k: v.cuda() for k, v in x.items()}


def gpu_forward(xd: dict, w, tiled: bool = False, query_order=None, fused: bool = True) -> dict:
    """Runs the precompute and the attention and returns every output on the
    CPU (fused: the one-pass precompute avq_assign_aggregate, else avq_assign
    then avq_aggregate; tiled: the App. B importance entry point;
    query_order: the ordered entry point, with Y returned in query order)."""
    if fused:
        par, code, packed, counts, Vbar = avq.assign_aggregate(xd["K"], xd["V"], xd["Cp"],
                                                               xd["Cc"], sums=True)
    else:
        par, code = avq.assign(xd["K"], xd["Cp"], xd["Cc"])
        packed, counts, Vbar = avq.aggregate(xd["V"], code, w.M0, w.Ch, sums=True)
    order = None if query_order is None else torch.as_tensor(query_order, dtype=torch.int32).cuda()
    Y, topp, imp = avq.attention_fwd(xd["Q"], xd["Cp"], xd["Cc"], packed, w.P, w.block_q,
                                     debug=True, tiled_importance=tiled, query_order=order)
    if order is not None:
        Y = Y[:, :, order.long()]
    torch.cuda.synchronize()
    out = dict(parent_idx=par, code_idx=code, Vbar=Vbar, packed=packed, counts=counts, Y=Y,
               topp=topp, importance=imp)
    return {k: v.cpu() for k, v in out.items()}


def unpack_packed(pk: np.ndarray, M0: int, Ch: int, d: int, dtype: str):
    """Packed aggregates [B, H, bytes] -> (means [B, H, Mtot, d] float64,
    n [B, H, Mtot], ln n [B, H, Mtot], padding dict).

    Layout: octets of 8 codes; the parent octets (padded to a multiple of 8
    octets), then ceil(Ch/8) child octets per parent, then one empty octet.
    Means [n_oct][d][8] in the storage dtype, then info [n_oct][16] fp32
    (n, then ln n)."""
    B, H, E = pk.shape
    PO, CO = -(-M0 // 64) * 8, -(-Ch // 8)
    n_oct = PO + M0 * CO + 1
    esz = 2 if dtype == "bf16" else 4
    info_off = n_oct * 8 * d * esz
    assert E == info_off + n_oct * 64
    raw = np.ascontiguousarray(pk[..., :info_off])
    if dtype == "bf16":
        bits = raw.view(np.uint16).astype(np.uint32) << 16
        vals = bits.view(np.float32)
    else:
        vals = raw.view(np.float32)
    vals = vals.astype(np.float64).reshape(B, H, n_oct, d, 8).transpose(0, 1, 2, 4, 3)
    info = np.ascontiguousarray(pk[..., info_off:]).view(np.float32).reshape(B, H, n_oct, 16)
    par = vals[:, :, :PO].reshape(B, H, PO * 8, d)
    ch = vals[:, :, PO:PO + M0 * CO].reshape(B, H, M0, CO * 8, d)
    means = np.concatenate([par[:, :, :M0], ch[:, :, :, :Ch].reshape(B, H, M0 * Ch, d)], axis=2)
    pn = info[:, :, :PO, :8].reshape(B, H, PO * 8)
    pl = info[:, :, :PO, 8:].reshape(B, H, PO * 8)
    cn = info[:, :, PO:PO + M0 * CO, :8].reshape(B, H, M0, CO * 8)
    cl = info[:, :, PO:PO + M0 * CO, 8:].reshape(B, H, M0, CO * 8)
    n = np.concatenate([pn[:, :, :M0], cn[:, :, :, :Ch].reshape(B, H, -1)], axis=2)
    ln = np.concatenate([pl[:, :, :M0], cl[:, :, :, :Ch].reshape(B, H, -1)], axis=2)
    pad = dict(
        means=np.concatenate([par[:, :, M0:].reshape(B, H, -1), ch[:, :, :, Ch:].reshape(B, H, -1),
                              vals[:, :, -1].reshape(B, H, -1)], axis=2),
        n=np.concatenate([pn[:, :, M0:], cn[:, :, :, Ch:].reshape(B, H, -1), info[:, :, -1, :8]],
                         axis=2),
        ln=np.concatenate([pl[:, :, M0:], cl[:, :, :, Ch:].reshape(B, H, -1), info[:, :, -1, 8:]],
                          axis=2))
    return means, n, ln, pad


class Report(dict):
    def line(self):
        return ", ".join(f"{k}={v}" for k, v in self.items())


def check_assign(x, w, g, o) -> tuple:
    """Certified-exact comparison of parent_idx / code_idx; every differing
    (uncertified) decision must be a valid choice within the bound."""
    K, Cp, Cc = oracle.f64(x["K"]), oracle.f64(x["Cp"]), oracle.f64(x["Cc"])
    d = w.d
    knorm = np.linalg.norm(K, axis=-1)
    cmax = np.linalg.norm(Cp, axis=-1).max(axis=-1)[None, :, None]  # per head
    err_p = gamma(d) * (cmax ** 2 + 2 * knorm * cmax) + U * (o["d_parent"] + cmax ** 2
                                                           + 2 * knorm * cmax)
    par_margin = o["d_parent2"] - o["d_parent"]
    par_cert = par_margin > 2 * 2 * err_p
    gp, gc = g["parent_idx"].numpy(), g["code_idx"].numpy()
    op, oc = o["parent_idx"], o["code_idx"]
    bad = par_cert & (gp != op)
    assert not bad.any(), f"{bad.sum()} certified parent decisions differ, e.g. at {np.argwhere(bad)[:5]}"
    if w.Ch == 0:
        return _check_flat_assign(K, Cp, w, gp, gc, op, err_p, par_cert)

    # child compare: bound both the direct form and ||c||^2 - 2 k.c (bf16)
    cn = np.maximum(np.linalg.norm(Cc, axis=-1).max(axis=(-1, -2)),
                    np.linalg.norm(Cp, axis=-1).max(axis=-1))[None, :, None]
    err_x = (gamma(d) + U) * (cn ** 2 + 2 * knorm * cn)
    err_c = 2 * err_x + gamma(d + 1) * (o["d_child"] + o["d_parent"]) + 1e-30
    move_cert = np.abs(o["d_child"] - o["d_parent"]) > 2 * err_c
    child_cert = (o["d_child2"] - o["d_child"]) > 2 * (2 * err_x + gamma(d + 1) * (
        o["d_child"] + o["d_child2"]))
    code_cert = par_cert & move_cert & (child_cert | (oc < w.M0))
    bad = code_cert & (gc != oc)
    assert not bad.any(), f"{bad.sum()} certified code decisions differ, e.g. at {np.argwhere(bad)[:5]}"

    # Uncertified differences must be valid choices within the bound.
    diff = (gc != oc) | (gp != op)
    for b, h, j in np.argwhere(diff):
        k = K[b, h, j]
        dp = ((Cp[h] - k) ** 2).sum(-1)
        assert dp[gp[b, h, j]] <= dp.min() + 4 * err_p[b, h, j], "invalid parent choice"
        p = gp[b, h, j]
        dc = ((Cc[h, p] - k) ** 2).sum(-1)
        dpar = dp[p]
        tol = 4 * err_x[b, h, j] + 4 * gamma(d + 1) * (dpar + dc.max())
        if gc[b, h, j] >= w.M0:
            cc = gc[b, h, j] - w.M0
            assert cc // w.Ch == p
            assert dc[cc % w.Ch] <= min(dc.min(), dpar) + tol
        else:
            assert gc[b, h, j] == p
            assert dpar <= dc.min() + tol
    rep = Report(keys=int(diff.size), uncertified=int((~code_cert).sum()),
                 differing=int(diff.sum()), heads_on_gpu_codes=int(diff.any(axis=-1).sum()),
                 moved_frac=round(float((oc >= w.M0).mean()), 4))
    return rep


def _check_flat_assign(K, Cp, w, gp, gc, op, err_p, par_cert) -> tuple:
    """Flat codebook: the code is the parent, exactly; an uncertified parent
    that differs from the oracle's must be within the bound of the nearest."""
    np.testing.assert_array_equal(gc, gp)
    diff = gp != op
    for b, h, j in np.argwhere(diff):
        dp = ((Cp[h] - K[b, h, j]) ** 2).sum(-1)
        assert dp[gp[b, h, j]] <= dp.min() + 4 * err_p[b, h, j], "invalid parent choice"
    rep = Report(keys=int(diff.size), uncertified=int((~par_cert).sum()),
                 differing=int(diff.sum()), heads_on_gpu_codes=int(diff.any(axis=-1).sum()),
                 moved_frac=0.0)
    return rep


def check_aggregate(x, w, g, o) -> Report:
    """Counts exact; Vbar within the fp32 summation bound (o: the oracle on the
    codes the GPU compared against, see oracle_on_gpu_codes)."""
    gn, gV = g["counts"].numpy(), g["Vbar"].numpy()
    on, oV = o["counts"], o["Vbar"]
    np.testing.assert_array_equal(gn, on)
    # |fl(sum) - sum| <= gamma_(n-1) sum |v| for each element; |V| aggregated by the oracle
    absV, _ = oracle.aggregate(np.abs(oracle.f64(x["V"])), o["parent_idx"], o["code_idx"], w.M0,
                               w.Ch)
    tol = gamma(np.maximum(on, 1))[..., None] * absV + 1e-30
    err = np.abs(gV.astype(np.float64) - oV)
    assert (err <= tol).all(), f"Vbar error {err.max()} above bound"
    assert (gn[..., :w.M0].sum(-1) == w.N).all()
    # Packed aggregates: means fl(fl(sum) * fl(1/n)) rounded to the storage
    # dtype; n exact; ln n within a few ulp; empty codes and padding slots
    # exactly 0 (means, n) and -inf (ln n).
    means, n_pk, ln_pk, pad = unpack_packed(g["packed"].numpy(), w.M0, w.Ch, w.d, w.dtype)
    assert (pad["means"] == 0).all(), "padding means of the packed aggregates are not zero"
    assert (pad["n"] == 0).all() and np.isneginf(pad["ln"]).all(), "padding info is not empty"
    np.testing.assert_array_equal(n_pk, on.astype(np.float32))
    nz = on > 0
    ln_err = np.abs(ln_pk.astype(np.float64) - np.log(np.maximum(on, 1)))
    assert (ln_err[nz] <= 8 * U * np.log(np.maximum(on, 2))[nz] + 1e-7).all(), \
        "ln n of the packed aggregates is off"
    assert np.isneginf(ln_pk[~nz]).all()
    n = np.maximum(on, 1)[..., None]
    omean = oV / n
    r_store = 2.0 ** -8 if w.dtype == "bf16" else U
    tol_m = tol / n + (3 * U + r_store) * np.abs(omean) + 1e-30
    err_m = np.abs(means - omean)
    assert (err_m <= tol_m).all(), f"mean error {err_m.max()} above bound"
    assert (means[on == 0] == 0).all(), "mean of an empty code is not zero"
    return Report(max_vbar_err=float(err.max()), max_mean_err=float(err_m.max()))


def importance_eps(x, w, o) -> float:
    Q, Cp = oracle.f64(x["Q"]), oracle.f64(x["Cp"])
    qmax = np.linalg.norm(Q, axis=-1).max()
    cmax = np.linalg.norm(Cp, axis=-1).max()
    S = np.einsum("bhnd,hmd->bhnm", Q[:, :, :64], Cp)
    spread = float((S.max(-1) - S.min(-1)).max()) * 1.5
    # the kernel evaluates exp2((S + ln n) log2 e - m - log2 Z): the logit sum
    # starts at ln n (gamma_d ln N more), and the shift m + log2 Z (|m| at most
    # about 1.5 max|S| + log2 N + the lazy margin) is rounded once more
    logN = math.log(max(w.N, 2))
    shift = 1.5 * qmax * cmax + logN / math.log(2) + 16
    return (4 * gamma(w.d) * qmax * cmax + gamma(w.d) * logN + 2 * U * (spread + 8)
            + 2 * U * shift + 2 * gamma(w.M0 + w.block_q))


def check_topp(x, w, g, o, tile_mask) -> tuple:
    """Importance within eps_w; top-P sets certified-exact; the order of
    topp_idx canonical. Returns the mask of tiles whose selection differs from
    the oracle's (uncertified, valid alternatives) and a report.

    Order: the kernel lists its selection by its own importance, descending,
    lowest index first among equal values; that is checked exactly against
    the importance it returns. Against the oracle, every certified cut point
    of the oracle's order (a gap between ranks k and k+1 above the bound) must
    split the kernel's list into the same two sets."""
    eps = importance_eps(x, w, o)
    T = w.n_tiles
    differ = np.zeros((w.B, w.H, T), bool)
    gw, ow = g["importance"].numpy().astype(np.float64), o["importance"]
    gt, ot = g["topp"].numpy(), o["selection"]
    rep = Report(tiles=int(tile_mask.sum()), uncertified=0, differing=0, cut_points=0,
                 eps_w=float(f"{eps:.3g}"))
    scale = ow.sum(-1, keepdims=True)  # = tile size
    bad = tile_mask[..., None] & ~(np.abs(gw - ow) <= eps * ow + 1e-6 * eps * scale)
    assert not bad.any(), (f"importance off at {np.argwhere(bad)[:3]}: max rel "
                           f"{np.max(np.abs(gw - ow)[bad] / np.maximum(ow[bad], 1e-30))}")
    empty = (o["counts"][..., :w.M0] == 0)[:, :, None, :]
    assert (gw[np.broadcast_to(empty, gw.shape) & tile_mask[..., None]] == 0).all(), \
        "empty parents must have exactly zero importance"
    if w.P == 0:
        return differ, rep
    # the kernel's own canonical order, exactly
    gsel = np.take_along_axis(g["importance"].numpy(), gt.astype(np.int64), -1)
    desc = gsel[..., :-1] > gsel[..., 1:]
    tie = (gsel[..., :-1] == gsel[..., 1:]) & (gt[..., :-1] < gt[..., 1:])
    wrong = tile_mask[..., None] & ~(desc | tie)
    assert not wrong.any(), f"topp_idx not in canonical order at {np.argwhere(wrong)[:3]}"
    for b, h, t in np.argwhere(tile_mask):
        wt = ow[b, h, t]
        sc = scale[b, h, t, 0]
        order = np.lexsort((np.arange(w.M0), -wt))
        srt = wt[order]
        gs, os_ = set(gt[b, h, t].tolist()), set(ot[b, h, t].tolist())
        assert len(gs) == w.P, "selection has repeated parents"
        wP = srt[w.P - 1]
        wnext = srt[w.P] if w.P < w.M0 else -np.inf
        certified = (wP - wnext) > 2 * eps * wP + 2e-6 * eps * sc or w.P == w.M0
        if not certified:
            rep["uncertified"] += 1
        if gs == os_:
            cut = (srt[:w.P - 1] - srt[1:w.P]) > 2 * eps * srt[:w.P - 1] + 2e-6 * eps * sc
            for k in np.flatnonzero(cut):
                assert set(gt[b, h, t, :k + 1].tolist()) == set(order[:k + 1].tolist()), (
                    f"topp_idx order differs from the oracle's at a certified rank {k}, "
                    f"tile {(b, h, t)}")
            rep["cut_points"] += int(cut.sum())
            continue
        assert not certified, f"certified top-P set differs at tile {(b, h, t)}"
        rep["differing"] += 1
        differ[b, h, t] = True
        # a valid alternative: nothing left out beats anything taken by more than the bound
        taken = np.array(sorted(gs))
        left = np.setdiff1d(np.arange(w.M0), taken)
        assert wt[taken].min() >= wt[left].max() * (1 - 2 * eps) - 2e-6 * eps * sc, (
            f"invalid top-P choice at tile {(b, h, t)}")
    return differ, rep


def check_output(x, w, g, o, tile_mask) -> Report:
    """Per row ||Y - Y*||_inf / ||Y*||_inf within the dtype's tolerance on every
    row of every compared tile."""
    tol = TOL_Y[w.dtype]
    gY = g["Y"].float().numpy().astype(np.float64)
    oY = o["Y"]
    rows = np.repeat(tile_mask, w.block_q, axis=-1)[..., :w.N]
    assert np.isfinite(gY).all(), "non-finite output"
    assert np.isfinite(oY[rows]).all()
    num = np.abs(gY - oY).max(-1)
    den = np.abs(oY).max(-1)
    rel = np.where(rows, num / np.maximum(den, 1e-30), 0.0)
    worst = np.unravel_index(np.argmax(rel), rel.shape)
    assert rel.max() <= tol, f"max row error {rel.max():.3g} > {tol} at {worst}"
    rel_rows = rel[rows]
    fro = np.linalg.norm((gY - oY)[rows]) / np.linalg.norm(oY[rows])
    return Report(rows=int(rows.sum()), max_rel=float(f"{rel.max():.3g}"),
                  median_rel=float(f"{np.median(rel_rows):.3g}"), frob_rel=float(f"{fro:.3g}"))


def oracle_on_gpu_codes(x, w, g, mask, recovered, importance_tile) -> dict:
    """The oracle's aggregates, importance, top-P and output computed from the
    GPU's codes (its certification distances are not needed downstream)."""
    gp = g["parent_idx"].numpy().astype(np.int32)
    gc = g["code_idx"].numpy().astype(np.int32)
    Vbar, counts = oracle.aggregate(x["V"], gp, gc, w.M0, w.Ch)
    if importance_tile is None:
        imp = oracle.importance(x["Q"], x["Cp"], counts, w.Ch, w.block_q, mask)
    else:
        imp = oracle.importance_tiled(x["Q"], x["Cp"], counts, w.Ch, w.block_q, importance_tile,
                                      mask)
    sel = oracle.topp(imp, w.P, mask)
    Y, zr = oracle.output(x["Q"], x["Cp"], x["Cc"], Vbar, counts, sel, w.block_q, recovered,
                          mask)
    return dict(parent_idx=gp, code_idx=gc, Vbar=Vbar, counts=counts, importance=imp,
                selection=sel, Y=Y, zratio=zr)


def compare(x, w, tiles_per_head=None, seed=0, recovered=True, tiled=False,
            query_order=None, fused=True) -> dict:
    """Runs GPU and oracle on the same inputs and checks every output.

    tiles_per_head: number of query tiles per head evaluated by the oracle
    (None: all). The first and last tile are always included. tiled: the
    App. B importance on both sides (tiles of avq.IMPORTANCE_TILE parents).
    query_order: the GPU takes the queries in this order; the oracle gets Q
    with its rows permuted the same way, and the GPU's Y is compared in that
    order. fused: which precompute the GPU runs (see gpu_forward)."""
    T = w.n_tiles
    mask = np.ones((w.B, w.H, T), np.uint8)
    if tiles_per_head is not None and tiles_per_head < T:
        rng = np.random.default_rng(seed)
        mask[:] = 0
        for b in range(w.B):
            for h in range(w.H):
                pick = rng.choice(T, tiles_per_head, replace=False)
                mask[b, h, pick] = 1
                mask[b, h, [0, T - 1]] = 1
    g = gpu_forward(to_gpu(x), w, tiled, query_order, fused)
    if query_order is not None:
        x = dict(x, Q=x["Q"][:, :, torch.as_tensor(query_order, dtype=torch.long)].contiguous())
    itile = avq.IMPORTANCE_TILE if tiled else None
    o = oracle.forward(x["Q"], x["K"], x["V"], x["Cp"], x["Cc"], w.P, w.block_q,
                       recovered=recovered, tile_mask=mask, importance_tile=itile)
    ra = check_assign(x, w, g, o)
    if ra["differing"]:
        # uncertified codes went the other way: follow the GPU's codes downstream
        o = oracle_on_gpu_codes(x, w, g, mask, recovered, itile)
    rg = check_aggregate(x, w, g, o)
    tmask = mask.astype(bool)
    differ, rt = check_topp(x, w, g, o, tmask)
    assert rt["differing"] <= max(1, 0.01 * rt["tiles"]), "too many differing top-P sets"
    if differ.any():
        # tiles whose (uncertified) selection differs: the oracle's output on
        # the GPU's selection
        sel = np.array(o["selection"], copy=True)
        sel[differ] = g["topp"].numpy()[differ]
        Yf, _ = oracle.output(x["Q"], x["Cp"], x["Cc"], o["Vbar"], o["counts"], sel, w.block_q,
                              recovered, differ.astype(np.uint8))
        rows = np.repeat(differ, w.block_q, axis=-1)[..., :w.N]
        o = dict(o, Y=np.where(rows[..., None], Yf, o["Y"]))
    ry = check_output(x, w, g, o, tmask)
    ry["rows_on_gpu_selection"] = int(np.repeat(differ, w.block_q, axis=-1)[..., :w.N].sum())
    return dict(assign=ra, aggregate=rg, topp=rt, output=ry, gpu=g, oracle=o)
