"""Plant plausible mistakes in copies of the oracle (on the CPU) and check that
the pins catch every one of them.

Each mutant is a textual substitution in oracle/sim_oracle.c, compiled into a
temporary library; the committed oracle is never modified.  A mutant that
passes every pin would mean the pins could not tell that mistake from the
paper's definition."""
import os
import sys
import tempfile

import pytest

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import oracle  # noqa: E402
import oracle_pins as P  # noqa: E402

MUTANTS = {
    "max_is_min": ("return a < b ? b : a;", "return a < b ? a : b;"),
    "ties_to_highest_group": ("F[g * max_stages + 0] < F[gs * max_stages + 0]",
                              "F[g * max_stages + 0] <= F[gs * max_stages + 0]"),
    "reject_at_deadline": ("if (prev > deadline)", "if (prev >= deadline)"),
    "dispatch_on_last_stage": ("F[g * max_stages + 0] < F[gs * max_stages + 0]",
                               "F[g * max_stages + max_stages - 1] < F[gs * max_stages + max_stages - 1]"),
    "clamped_dispatch_key": ("F[g * max_stages + 0] < F[gs * max_stages + 0]",
                             "oracle_max(F[g * max_stages + 0], ti) < oracle_max(F[gs * max_stages + 0], ti)"),
    "first_hosting_group": ("if (gs < 0 || F[g * max_stages + 0] < F[gs * max_stages + 0]) gs = g;",
                            "if (gs < 0) gs = g;"),
    "no_queueing": ("f[s] = oracle_max(prev, F[gs * max_stages + s]) + lat;", "f[s] = prev + lat;"),
    "no_service_time": ("f[s] = oracle_max(prev, F[gs * max_stages + s]) + lat;",
                        "f[s] = oracle_max(prev, F[gs * max_stages + s]);"),
    "stage0_state_everywhere": ("f[s] = oracle_max(prev, F[gs * max_stages + s]) + lat;",
                                "f[s] = oracle_max(prev, F[gs * max_stages + 0]) + lat;"),
    "chain_starts_at_zero": ("double prev = ti;", "double prev = 0.0;"),
    "stage_table_transposed": ("stage_lat[((int64_t)m * n_configs + c) * max_stages + s]",
                               "stage_lat[((int64_t)c * n_models + m) * max_stages + s]"),
    "commit_when_rejected": ("if (prev > deadline) {\n        out = -1.0;",
                             "for (int32_t s = 0; s < S; ++s) F[gs * max_stages + s] = f[s];\n"
                             "      if (prev > deadline) {\n        out = -1.0;"),
    "update_stage0_only": ("for (int32_t s = 0; s < S; ++s) F[gs * max_stages + s] = f[s];\n        if (model_served_out)",
                           "F[gs * max_stages + 0] = f[0];\n        if (model_served_out)"),
    "slo_additive": ("slo[m] = slo_scale * d_single[m];", "slo[m] = slo_scale + d_single[m];"),
    "deadline_from_free_time": ("const double deadline = ti + slo[m];",
                                "const double deadline = F[gs * max_stages + 0] + slo[m];"),
    "finsum_of_stage0": ("fin_sum += bits_of(prev);", "fin_sum += bits_of(f[0]);"),
    "accept_bit_shifted": ("word |= (uint64_t)1 << (i & 63);", "word |= (uint64_t)1 << ((i + 1) & 63);"),
    "last_word_not_folded": ("if ((i & 63) == 63 || i == n - 1)", "if ((i & 63) == 63)"),
}


def _pins_fail(lib):
    failed = []
    for pin in P.ALL_PINS:
        try:
            pin(lib)
        except (AssertionError, ValueError):
            failed.append(pin.__name__)
    return failed


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name):
    old, new = MUTANTS[name]
    with open(oracle.SRC_PATH) as f:
        src = f.read()
    assert src.count(old) >= 1, f"mutation site for {name} not found"
    mutated = src.replace(old, new, 1)
    with tempfile.TemporaryDirectory() as d:
        path = os.path.join(d, f"mut_{name}.c")
        with open(path, "w") as f:
            f.write(mutated)
        so = oracle.build(path, os.path.join(d, f"libmut_{name}.so"))
        failed = _pins_fail(oracle.OracleLib(so))
    assert failed, f"no pin catches mutant {name}"
