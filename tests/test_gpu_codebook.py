"""GPU parity of the codebook update (App. A): avq_assign, then avq_aggregate
on the keys, then avq_codebook_update, against the oracle's assignment, key
aggregates and fp64 update on the same seeded inputs.

Every head is compared: certified assignment decisions must match the
oracle's; an uncertified one that went the other way must be a valid choice,
and the oracle then aggregates the keys on the GPU's codes (tests/parity.py).
Bounds,
u = 2^-24: the batch key sums carry gamma_n sum|k| per element (fp32 sums in
bucket order) and the batch reduction gamma_B; S' = fma(lambda, S, (1-lambda)
s) adds 2u |S'|; N' is exact up to 2u |N'|; each mean M = S'/N' adds 2u; the
projection adds 8u (sum_c |M_c| + (Ch+1) |C_p|) for delta and its division;
the stored codewords add the rounding to their type (2^-8 for bf16).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_12789_amd import inputs
from tests import parity

pytestmark = pytest.mark.gpu
U = 2.0 ** -24


def small(**kw):
    base = dict(name="ema", B=2, H=3, N=1000, d=64, M0=40, Ch=4, P=0, block_q=128,
                dtype="bf16", sigma_c=0.1, sigma_k=0.05, seed=2)
    base.update(kw)
    return inputs.Workload(**base)


def ema_state(w, seed):
    """A positive EMA state: masses in [0.5, 50), sums = mass * (codeword + noise)."""
    rng = np.random.default_rng(seed)
    Mtot = w.Mtot
    N0 = rng.uniform(0.5, 50.0, (w.H, Mtot)).astype(np.float32)
    S0 = (N0[..., None] * rng.standard_normal((w.H, Mtot, w.d))).astype(np.float32)
    return S0, N0


def run(w, lam, x=None, seed=0):
    from paper_2607_12789_amd import avq
    x = inputs.generate(w) if x is None else x
    xd = parity.to_gpu(x)
    par, code = avq.assign(xd["K"], xd["Cp"], xd["Cc"])
    _, counts, sums = avq.aggregate(xd["K"], code, w.M0, w.Ch, sums=True)
    S0, N0 = ema_state(w, seed)
    S = torch.from_numpy(S0).cuda()
    Nm = torch.from_numpy(N0).cuda()
    Cp, Cc = avq.codebook_update(sums, counts, S, Nm, w.M0, w.Ch, lam, dtype=w.torch_dtype)
    torch.cuda.synchronize()
    g = dict(parent_idx=par.cpu(), code_idx=code.cpu(), S=S.cpu().numpy().astype(np.float64),
             N=Nm.cpu().numpy().astype(np.float64), Cp=Cp.float().cpu().numpy().astype(np.float64),
             Cc=Cc.float().cpu().numpy().astype(np.float64))

    a = oracle.assign(x["K"], x["Cp"], x["Cc"])
    # certified decisions must match; any uncertified one that went the other
    # way must be valid, and the oracle then aggregates on the GPU's codes
    parity.check_assign(x, w, g, a)
    a = dict(a, parent_idx=g["parent_idx"].numpy().astype(np.int32),
             code_idx=g["code_idx"].numpy().astype(np.int32))
    o_sums, o_counts = oracle.aggregate(x["K"], a["parent_idx"], a["code_idx"], w.M0, w.Ch)
    # the entry point takes lambda as fp32: the oracle uses that same value
    lam32 = float(np.float32(lam))
    S2, N2, oCp, oCc = oracle.codebook_update(o_sums, o_counts, S0, N0, w.M0, w.Ch, lam32)
    abs_sums, _ = oracle.aggregate(np.abs(oracle.f64(x["K"])), a["parent_idx"], a["code_idx"],
                                   w.M0, w.Ch)
    o = dict(a, S=S2, N=N2, Cp=oCp, Cc=oCc, sums=o_sums, counts=o_counts, abs_sums=abs_sums)
    return x, g, o


def check(w, lam, x, g, o):
    heads = np.ones(w.H, bool)  # every head (the oracle follows the GPU's codes)
    n = o["counts"].astype(np.float64)  # [B, H, Mtot]
    gam = lambda k: k * U / (1 - k * U)
    err_s = (gam(np.maximum(n, 1))[..., None] * o["abs_sums"]).sum(0) \
        + gam(w.B) * np.abs(o["sums"]).sum(0)                    # [H, Mtot, d]
    S2, N2 = o["S"], o["N"]
    # 1 - lambda is rounded to fp32 once more on the GPU
    s_tot, n_tot = o["sums"].sum(0), n.sum(0)
    err_S = (1 - lam) * (err_s + 2 * U * np.abs(s_tot)) + 2 * U * np.abs(S2) + 1e-30
    err_N = 2 * U * ((1 - lam) * n_tot + N2) + 1e-30
    np.testing.assert_array_less(np.abs(g["S"] - S2)[heads], err_S[heads] * 1.0001)
    np.testing.assert_array_less(np.abs(g["N"] - N2)[heads], err_N[heads] * 1.0001)
    M = S2 / N2[..., None]
    err_M = (err_S + np.abs(S2) * err_N[..., None] / N2[..., None]) / N2[..., None] \
        + 4 * U * np.abs(M)
    r_store = 2.0 ** -8 if w.dtype == "bf16" else U
    pM, pE = M[:, :w.M0], err_M[:, :w.M0]
    tol_p = pE + r_store * np.abs(o["Cp"]) + 1e-30
    errp = np.abs(g["Cp"] - o["Cp"])
    assert (errp[heads] <= tol_p[heads]).all(), f"parent codeword error {errp[heads].max()}"
    if w.Ch == 0:
        return
    cM = M[:, w.M0:].reshape(w.H, w.M0, w.Ch, w.d)
    cE = err_M[:, w.M0:].reshape(w.H, w.M0, w.Ch, w.d)
    proj = (8 * U * (np.abs(cM).sum(2) + (w.Ch + 1) * np.abs(pM)) + cE.sum(2)
            + (w.Ch + 1) * pE)[:, :, None, :]
    tol_c = cE + proj + r_store * np.abs(o["Cc"]) + 1e-30
    errc = np.abs(g["Cc"] - o["Cc"])
    assert (errc[heads] <= tol_c[heads]).all(), f"child codeword error {errc[heads].max()}"
    # the constraint holds up to the stored rounding
    if w.dtype == "f32":
        gap = np.abs(g["Cc"].mean(2) - g["Cp"])
        assert (gap[heads] <= (tol_c.max(2) + tol_p)[heads]).all()


CASES = {
    "bf16_ch4": (small(), 0.9),
    "f32_ch8_d128": (small(dtype="f32", Ch=8, d=128, M0=30), 0.99),
    "f32_lambda_small": (small(dtype="f32", Ch=4, M0=32), 0.1),
    "bf16_ch16": (small(Ch=16, M0=20, N=1500), 0.5),
    "f32_flat": (small(dtype="f32", Ch=0, M0=64), 0.8),
    "bf16_ch1_b1": (small(Ch=1, B=1, M0=70), 0.3),
    "f32_lambda_one": (small(dtype="f32", Ch=2, M0=50), 1.0),
    "bf16_m0_512_d128": (small(M0=512, Ch=8, d=128, N=4096, B=1, H=2), 0.95),
    "f32_ch16_d64": (small(dtype="f32", Ch=16, M0=20, N=1500), 0.75),
}


@pytest.mark.parametrize("name", list(CASES))
def test_codebook_update(name):
    w, lam = CASES[name]
    print(f"[codebook_update] {name}: {w.describe()} lambda={lam}", flush=True)
    x, g, o = run(w, lam)
    check(w, lam, x, g, o)


def test_codebook_update_lambda_one_keeps_the_state():
    """lambda = 1: S and N are left exactly as they were."""
    w = small(dtype="f32", Ch=4, M0=20, N=300)
    _, g, _ = run(w, 1.0, seed=5)
    S0, N0 = ema_state(w, 5)
    np.testing.assert_array_equal(g["S"], S0.astype(np.float64))
    np.testing.assert_array_equal(g["N"], N0.astype(np.float64))
