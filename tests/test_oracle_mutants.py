"""Plants plausible mistakes in copies of the oracle (on the CPU) and checks
that the pins in ``test_oracle_pins.py`` catch every one of them.

Each mutant is a one-line textual edit of ``oracle/avq_oracle.c`` compiled
into a temporary library; the pins are then run against it and at least one
must fail. The real oracle is restored afterwards.
"""
import contextlib
import subprocess
from pathlib import Path

import pytest

import oracle
from tests import test_oracle_pins as pins

SRC = Path(oracle.__file__).resolve().parent / "avq_oracle.c"

# (name, original text, mutated text)
MUTANTS = [
    ("denominator drops the count weight",
     "Z += A * (double)n[a];", "Z += A;"),
    ("child moves on equal distance",
     "code_idx[t] = (dc < dbest)", "code_idx[t] = (dc <= dbest)"),
    ("parent ties go to the highest index",
     "if (dist < dbest) {\n        dsecond = dbest;", "if (dist <= dbest) {\n        dsecond = dbest;"),
    ("importance drops the count weight",
     "if (n[a] > 0) wt[a] += (double)n[a] * exp(S[a] - mu) / Z;",
     "if (n[a] > 0) wt[a] += exp(S[a] - mu) / Z;"),
    ("top-P takes the smallest importance",
     "if (best < 0 || wr[a] > wr[best]) best = a;", "if (best < 0 || wr[a] < wr[best]) best = a;"),
    ("correction sign flipped",
     "double dA = exp(Tc[k * Ch + c] - mu) - Ap;", "double dA = Ap - exp(Tc[k * Ch + c] - mu);"),
    ("recovered logit uses the first child only",
     "R[k] = recovered ? mean / Ch : S[p];", "R[k] = recovered ? Tc[k * Ch] : S[p];"),
    ("child code index transposed",
     "(M0 + best * Ch + cbest)", "(M0 + cbest * M0 + best)"),
    ("parent rows only count keys that stayed",
     "      n[p] += 1;\n", "      if (code_idx[t] < M0) n[p] += 1;\n"),
    ("empty children not masked in the correction",
     "          if (n[code] == 0) continue;\n          double dA", "          double dA"),
    ("importance uses an unnormalised weight",
     "wt[a] += (double)n[a] * exp(S[a] - mu) / Z;", "wt[a] += (double)n[a] * exp(S[a] - mu);"),
    ("child logits against the parent codeword",
     "double v = dot(q, Cc + (((long long)h * M0 + p) * Ch + c) * d, d);",
     "double v = dot(q, Cp + ((long long)h * M0 + p) * d, d);"),
    ("tiled importance without the count extrapolation",
     "double zt = (double)N / (double)seen * zsum;", "double zt = zsum;"),
    ("tiled importance counts the keys of the current tile only",
     "for (int a0 = 0; a0 < M0; a0 += tile_c) {\n", "for (int a0 = 0; a0 < M0; a0 += tile_c) {\n        seen = 0;\n"),
    ("tiled importance scales by the partial denominator of the tile alone",
     "if (n[a] > 0) zsum += (double)n[a] * exp(S[a] - mu);",
     "if (n[a] > 0) zsum = (double)n[a] * exp(S[a] - mu);"),
    ("projection ignores the child masses",
     "- delta / (Nema[rc] * sigma);", "- delta / (double)Ch;"),
    ("EMA adds the batch statistics at full weight",
     "Nema[r] = lambda * Nema[r] + (1.0 - lambda) * n;", "Nema[r] = lambda * Nema[r] + n;"),
    ("harmonic weight without the reciprocal",
     "sigma += 1.0 / Nema[(long long)h * Mtot + M0 + p * Ch + c];",
     "sigma += Nema[(long long)h * Mtot + M0 + p * Ch + c];"),
    ("constraint residual with the wrong sign",
     "double delta = -(double)Ch * cp[e];", "double delta = (double)Ch * cp[e];"),
]

PIN_CALLS = [
    lambda: pins.test_assign_matches_cdist(0),
    pins.test_assign_exact_ties_lowest_index,
    pins.test_aggregates_match_add_at_and_invariants,
    lambda: pins.test_importance_equals_per_key_attention_mass(32),
    lambda: pins.test_topp_matches_enumeration(3),
    pins.test_p0_is_vq_attention,
    lambda: pins.test_refined_direct_equals_per_key_replacement(2, 32),
    pins.test_refined_recovered_per_key_weights,
    pins.test_zero_queries_give_mean_value,
    pins.test_children_equal_parent_reduce_to_vq,
    pins.test_large_logits_stay_finite,
    pins.test_empty_far_children_do_not_poison,
    lambda: pins.test_tiled_importance_last_tile_is_exact(3),
    pins.test_tiled_importance_first_tile_closed_form,
    lambda: pins.test_tiled_importance_zero_queries(3),
    pins.test_codebook_update_keeps_the_constraint,
    lambda: pins.test_codebook_update_solves_the_weighted_least_squares(4),
    pins.test_codebook_update_ema_closed_form,
]


@contextlib.contextmanager
def mutant_library(tmp_path, old, new):
    src = SRC.read_text()
    assert src.count(old) == 1, f"mutation anchor not unique: {old!r}"
    mpath = tmp_path / "mutant.c"
    mpath.write_text(src.replace(old, new))
    so = tmp_path / "libmutant.so"
    subprocess.run(["gcc", "-O1", "-std=c99", "-fopenmp", "-fPIC", "-shared", str(mpath),
                    "-o", str(so), "-lm"], check=True)
    saved = oracle._load()
    oracle._lib = oracle.open_library(so)
    try:
        yield
    finally:
        oracle._lib = saved


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_mutant(tmp_path, name, old, new):
    caught = []
    with mutant_library(tmp_path, old, new):
        for call in PIN_CALLS:
            try:
                call()
            except (AssertionError, ValueError, FloatingPointError):
                caught.append(call)
                break
    assert caught, f"no pin fails for the mutant '{name}'"


# Mistakes planted in the oracle's capture (App. B, tab. tiled_capture), a
# Python function: each is a textual edit of its source, compiled in the
# oracle module's namespace and swapped in for the duration of the pins.
CAPTURE_MUTANTS = [
    ("best selection is the given selection",
     "best += mass[:, top].sum()", "best += mass[:, sel[b, h, t]].sum()"),
    ("best selection ranked per query instead of per tile",
     "best += mass[:, top].sum()", "best += np.sort(mass, axis=1)[:, mass.shape[1] - P:].sum()"),
    ("best selection ranked by key count",
     "top = np.argsort(-mass.sum(axis=0), kind=\"stable\")[:P]",
     "top = np.argsort(-onehot.sum(axis=0), kind=\"stable\")[:P]"),
    ("best selection takes the smallest masses",
     "top = np.argsort(-mass.sum(axis=0), kind=\"stable\")[:P]",
     "top = np.argsort(mass.sum(axis=0), kind=\"stable\")[:P]"),
    ("attention weights not normalised",
     "A /= A.sum(axis=1, keepdims=True)", "A = A"),
]

CAPTURE_PINS = [
    lambda: pins.test_capture_best_selection_by_enumeration(2),
    pins.test_capture_hand_worked,
    pins.test_capture_of_full_selection_is_one,
]


@pytest.mark.parametrize("name,old,new", CAPTURE_MUTANTS, ids=[m[0] for m in CAPTURE_MUTANTS])
def test_capture_pins_catch_mutant(monkeypatch, name, old, new):
    import inspect
    import textwrap
    src = textwrap.dedent(inspect.getsource(oracle.capture))
    assert src.count(old) == 1, f"mutation anchor not unique: {old!r}"
    ns = dict(vars(oracle))
    exec(compile(src.replace(old, new), "<capture mutant>", "exec"), ns)
    monkeypatch.setattr(oracle, "capture", ns["capture"])
    caught = []
    for call in CAPTURE_PINS:
        try:
            call()
        except (AssertionError, ValueError, IndexError):
            caught.append(call)
            break
    assert caught, f"no pin fails for the capture mutant '{name}'"


def test_capture_pins_pass_on_the_oracle():
    for call in CAPTURE_PINS:
        call()
