"""Plant plausible mistakes in copies of the search oracles and of the
dynamic-batching oracle (on the CPU) and check that the pins catch each one.

Python mutants are textual substitutions in oracle/greedy.py or oracle/alg2.py,
executed as a module of their own and put in place of the committed module
inside the pin modules (tests/test_oracle_search.py, test_oracle_greedy.py,
test_oracle_alg2.py) for the duration of one test.  C mutants are
substitutions in oracle/sim_oracle.c compiled into a temporary library and run
through the batching pins (tests/test_oracle_batching.py).  The committed
oracle is never modified.  A mutant that passes every pin would mean the pins
could not tell that mistake from the rule the paper states."""
import importlib.util
import inspect
import os
import sys
import tempfile

import pytest

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import oracle  # noqa: E402
import test_oracle_alg2 as PA  # noqa: E402
import test_oracle_batching as PB  # noqa: E402
import test_oracle_greedy as PG  # noqa: E402
import test_oracle_search as PS  # noqa: E402

ORACLE_DIR = os.path.dirname(oracle.SRC_PATH)

# Alg. 1 (beam k), the fast heuristic and the greedy loop (Sec. 4.2)
GREEDY_MUTANTS = {
    # two beam entries reaching the same replica set both kept
    "beam_no_dedup": ("if key in seen:\n                        continue",
                      "if False:\n                        continue"),
    # the k LEAST served selections kept
    "beam_topk_ascending": ("key=lambda i: (-scores[i], i))[:beam]", "key=lambda i: (scores[i], i))[:beam]"),
    # only the single best selection carried into the next step
    "beam_keeps_one": ("for i in order]", "for i in order[:1]]"),
    # the heuristic places the model with the FEWEST unserved requests
    "fast_least_unserved_model": ("if mstar is None or n_req[m] - ms[m] > n_req[mstar] - ms[mstar]:",
                                  "if mstar is None or n_req[m] - ms[m] < n_req[mstar] - ms[mstar]:"),
    # ... on the BUSIEST available group
    "fast_busiest_group": ("busy[g] < busy[gstar]", "busy[g] > busy[gstar]"),
    # unserved counted as served
    "fast_served_not_unserved": ("n_req[m] - ms[m] > n_req[mstar] - ms[mstar]", "ms[m] > ms[mstar]"),
    # the last simulated selection does not compete for the result
    "fast_last_not_scored": ("if served > best_served:\n            best_served = served",
                             "if served > best_served and len(steps) < 0:\n            best_served = served"),
    # greedy ties to the LAST candidate
    "greedy_ties_to_last": ("if scores[i] > scores[bi]:", "if scores[i] >= scores[bi]:"),
    # a group that already hosts the model offered again
    "candidates_rehost": ("if (int(host_mask[m]) >> g) & 1:\n                continue",
                          "if False:\n                continue"),
    # memory must stay strictly below the group's capacity
    "memory_strict": ("<= int(group_mem_mib[g])", "< int(group_mem_mib[g])"),
}

# Alg. 2 (Sec. 4.2): model buckets, device splits, pruning, partitions
ALG2_MUTANTS = {
    # buckets may span twice the latency threshold
    "threshold_widened": ("if d[order[end - 1]] - d[order[pos]] > threshold:",
                          "if d[order[end - 1]] - d[order[pos]] > 2.0 * threshold:"),
    # bucket order by id among equal latencies reversed
    "order_ties_reversed": ("key=lambda m: (d[m], m))", "key=lambda m: (d[m], -m))"),
    # the largest part of a device split never enumerated
    "splits_truncated": ("for x in range(1, left - (parts - 1) + 1):",
                         "for x in range(1, left - (parts - 1)):"),
    # remainder group on the SHALLOWEST pipeline of its size
    "remainder_shallowest": ("if last is None or cfg_stages[c2] > cfg_stages[last]:",
                             "if last is None or cfg_stages[c2] < cfg_stages[last]:"),
    # remainder group may be deeper than the bucket's configuration
    "remainder_any_depth": ("if int(cfg_devices[c2]) == rem and cfg_stages[c2] <= cfg_stages[c]:",
                            "if int(cfg_devices[c2]) == rem:"),
    # a placement scored by its best bucket instead of the sum over buckets
    "max_over_buckets": ('total += entry["served"]', 'total = max(total, entry["served"])'),
    # no pruning of unbalanced device splits
    "no_balance_pruning": ("if not (max(rhos) <= balance_ratio * min(rhos)):\n                    continue",
                           "if False:\n                    continue"),
    # bucket load not divided by the bucket's devices
    "load_per_bucket_not_per_device": ("rhos.append(load / float(H[b]))", "rhos.append(load)"),
    # the last group of a bucket dropped (only the equal groups)
    "remainder_dropped": ("            groups.append(last)\n", ""),
}

# dynamic batching (Sec. 6.5), oracle_simulate_job_batched in sim_oracle.c
BATCH_MUTANTS = {
    # the batch factor applied twice per stage
    "batch_factor_twice": ("const double lat_ = stage_lat[((int64_t)(m) * n_configs + c_) * max_stages + s_] * fac_;",
                           "const double lat_ = stage_lat[((int64_t)(m) * n_configs + c_) * max_stages + s_] * fac_ * fac_;"),
    # an idle group serves the model whose queue head arrived LAST
    "youngest_queue_head": ("(mc < 0 || q[m].idx[q[m].head] < q[mc].idx[q[mc].head])",
                            "(mc < 0 || q[m].idx[q[m].head] > q[mc].idx[q[mc].head])"),
    # a head that cannot meet its deadline runs anyway as a batch of one
    "no_head_drop": ("q[mc].head += 1; /* the head cannot meet its deadline: dropped */\n          continue;",
                     "b = 1;"),
    # an arrival runs at once even when every hosting group is busy
    "arrival_ignores_busy": ("if (((mask >> g) & 1u) && F[g * max_stages] <= t[i] &&",
                             "if (((mask >> g) & 1u) &&"),
    # the deadline of the batch taken from the request after the head
    "deadline_not_head": ("const double dl = t[hd] + slo[mc];",
                          "const double dl = t[q[mc].idx[q[mc].tail - 1]] + slo[mc];"),
    # an arrival that would miss its deadline is still served
    "arrival_no_drop": ("if (!(f[S - 1] > t[i] + slo[m])) {", "if (1) {"),
}


def _load_mutant(modname, old, new):
    """Module oracle.<modname> with `old` replaced by `new` once (relative
    imports resolve inside the committed oracle package)."""
    path = os.path.join(ORACLE_DIR, modname + ".py")
    with open(path) as f:
        src = f.read()
    assert src.count(old) >= 1, f"mutation site not found in {modname}.py: {old!r}"
    mutated = src.replace(old, new, 1)
    spec = importlib.util.spec_from_loader(f"oracle._mutant_{modname}", loader=None)
    mod = importlib.util.module_from_spec(spec)
    mod.__package__ = "oracle"
    exec(compile(mutated, f"<mutant of oracle/{modname}.py>", "exec"), mod.__dict__)
    return mod


def _calls(fn):
    """Argument tuples of a pin test function (its parametrize marks expanded;
    the olib fixture comes first)."""
    params = [p for p in inspect.signature(fn).parameters if p != "olib"]
    if not params:
        return [{}]
    for mark in getattr(fn, "pytestmark", []):
        if mark.name == "parametrize":
            names = [s.strip() for s in mark.args[0].split(",")]
            out = []
            for v in mark.args[1]:
                v = v if len(names) > 1 else (v,)
                out.append(dict(zip(names, v)))
            return out
    raise AssertionError(f"{fn.__name__}: parameters {params} without parametrize")


def _run_pins(modules, olib):
    """Names of the pin tests (in the given modules) that fail."""
    failed = []
    for mod in modules:
        for name, fn in sorted(vars(mod).items()):
            if not (name.startswith("test_") and callable(fn)):
                continue
            takes_lib = "olib" in inspect.signature(fn).parameters
            for kw in _calls(fn):
                try:
                    fn(olib, **kw) if takes_lib else fn(**kw)
                except (AssertionError, ValueError, KeyError, IndexError, TypeError, ZeroDivisionError):
                    failed.append(f"{mod.__name__}.{name}{kw or ''}")
    return failed


@pytest.mark.parametrize("name", sorted(GREEDY_MUTANTS))
def test_greedy_mutant_is_caught(name, olib, monkeypatch):
    mut = _load_mutant("greedy", *GREEDY_MUTANTS[name])
    for mod in (PS, PG, PA):
        monkeypatch.setattr(mod, "greedy", mut)
    failed = _run_pins((PS, PG), olib)
    assert failed, f"no pin catches greedy mutant {name}"


@pytest.mark.parametrize("name", sorted(ALG2_MUTANTS))
def test_alg2_mutant_is_caught(name, olib, monkeypatch):
    mut = _load_mutant("alg2", *ALG2_MUTANTS[name])
    monkeypatch.setattr(PA, "alg2", mut)
    failed = _run_pins((PA,), olib)
    assert failed, f"no pin catches Alg. 2 mutant {name}"


@pytest.mark.parametrize("name", sorted(BATCH_MUTANTS))
def test_batching_mutant_is_caught(name):
    old, new = BATCH_MUTANTS[name]
    with open(oracle.SRC_PATH) as f:
        src = f.read()
    assert src.count(old) >= 1, f"mutation site for {name} not found"
    mutated = src.replace(old, new, 1)
    with tempfile.TemporaryDirectory() as d:
        path = os.path.join(d, f"mut_{name}.c")
        with open(path, "w") as f:
            f.write(mutated)
        so = oracle.build(path, os.path.join(d, f"libmut_{name}.so"))
        failed = _run_pins((PB,), oracle.OracleLib(so))
    assert failed, f"no pin catches batching mutant {name}"


def test_committed_oracle_passes_every_pin(olib):
    """The harness itself: with nothing planted, no pin fails."""
    assert _run_pins((PS, PG, PA, PB), olib) == []
