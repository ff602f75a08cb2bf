"""A forward pass captured in a HIP graph and replayed.

The entry points enqueue kernels only (no memset, copy, allocation or host
wait), so once each has run eagerly on the device (which caches the device
attributes and kernel settings) a sequence of calls can be captured. Every
replay rewrites the outputs (zeroed before it), with eager forward passes on
other inputs and synchronisations between the replays, and is checked against
the eager pass: integers exactly, Y within the run-to-run rounding of the
value sums (their summation order within a code follows the LDS atomics that
bucket the keys).
"""
import dataclasses
import sys

import pytest
import torch

from paper_2607_12789_amd import avq, inputs

pytestmark = pytest.mark.gpu

CASES = {
    "bf16_d128": inputs.Workload("graph_bf16", B=2, H=2, N=700, d=128, M0=96, Ch=8, P=12,
                                 block_q=128),
    "f32_d64": inputs.Workload("graph_f32", B=1, H=2, N=500, d=64, M0=40, Ch=4, P=6, block_q=64,
                               dtype="f32"),
}


@pytest.mark.parametrize("name", list(CASES))
def test_forward_replayed_from_a_graph(name):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    w = CASES[name]
    print(f"\n[case] graph replay {name}: {w.describe()}", flush=True)
    sys.stdout.flush()
    x = {k: v.cuda() for k, v in inputs.generate(w).items()}
    other = {k: v.cuda() for k, v in inputs.generate(dataclasses.replace(w, seed=7)).items()}

    par, code, packed, counts, _ = avq.assign_aggregate(x["K"], x["V"], x["Cp"], x["Cc"])
    Y = avq.attention_fwd(x["Q"], x["Cp"], x["Cc"], packed, w.P, w.block_q)
    torch.cuda.synchronize()
    ref = {"par": par.clone(), "code": code.clone(), "counts": counts.clone(), "Y": Y.clone()}

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        avq.assign_aggregate(x["K"], x["V"], x["Cp"], x["Cc"], par, code, packed, counts)
        avq.attention_fwd(x["Q"], x["Cp"], x["Cc"], packed, w.P, w.block_q, Y=Y)

    for rep in range(3):
        for t in (par, code, packed, counts, Y):
            t.zero_()
        # eager work of the program between the replays
        _, _, pk2, _, _ = avq.assign_aggregate(other["K"], other["V"], other["Cp"], other["Cc"])
        avq.attention_fwd(other["Q"], other["Cp"], other["Cc"], pk2, w.P, w.block_q)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        print(f"  replay {rep}", flush=True)
        assert torch.equal(par, ref["par"]), f"replay {rep}: parent indices"
        assert torch.equal(code, ref["code"]), f"replay {rep}: codes"
        assert torch.equal(counts, ref["counts"]), f"replay {rep}: counts"
        torch.testing.assert_close(Y.float(), ref["Y"].float(), rtol=2e-3, atol=1e-5)
