"""Planted mistakes in the oracle must be caught by its pins.

Each case copies the oracle source, applies one plausible slip (a dropped
term, a flipped sign, a wrong index, a transposed operand, a wrong tie-break),
builds it with g++ into a temporary library and runs the pin suite's checks on
it: at least one must fail.  The mutated builds live only in a temporary
directory and are never used by anything else.
"""
import ctypes
import os
import subprocess

import numpy as np
import pytest

import oracle
from golden_io import load as load_golden, names as golden_names
from paper_2601_05109_amd import workloads as wl
from test_oracle_pins import (brute_force_rem, push_replay_ready, rem_certificate,
                              assert_routes_exhaustive, wide_range,
                              test_lpt_equals_srtf_when_deadlines_are_equal,
                              test_lpt_independent_futures_closed_form, test_stateful_routing_pins,
                              test_greedy_single_instance_prefix_sums,
                              test_greedy_identical_instances_round_robin,
                              test_priority_levels_partition_the_order,
                              test_srtf_independent_futures_closed_form,
                              test_weighted_against_quota_walk, test_weighted_rules,
                              test_weighted_whole_periods_are_proportional)

MUTATIONS = {
    "drop_est_term": ("if (__builtin_add_overflow(est_eff[v], best, &r)",
                      "if (__builtin_add_overflow(int64_t(0), best, &r)"),
    "done_not_zeroed": ("est_eff[v] = done[v] ? 0 : est[v];", "est_eff[v] = est[v];"),
    "slack_sign": ("slack[v] = (deadline[wf[v]] - now) - rem[v];",
                   "slack[v] = (deadline[wf[v]] - now) + rem[v];"),
    "slack_wrong_index": ("slack[v] = (deadline[wf[v]] - now) - rem[v];",
                          "slack[v] = (deadline[type[v] % (W ? W : 1)] - now) - rem[v];"),
    "penalty_inverted": ("inst_speed[i];\n      if (loc[v] >= 0 && loc[v] != i) c += mig;",
                         "inst_speed[i];\n      if (loc[v] >= 0 && loc[v] == i) c += mig;"),
    "penalty_dropped": ("inst_speed[i];\n      if (loc[v] >= 0 && loc[v] != i) c += mig;", "inst_speed[i];"),
    "division_transposed": ("int64_t c = inst_load[i] + (est[v] * 1000) / inst_speed[i];",
                            "int64_t c = inst_load[i] + (inst_speed[i] * 1000) / (est[v] + 1);"),
    "tie_to_highest": ("      if (c < best) { best = c; arg = int32_t(i); }\n    }\n    route[v] = arg;\n    cost[v] = best;\n  }",
                       "      if (c <= best) { best = c; arg = int32_t(i); }\n    }\n    route[v] = arg;\n    cost[v] = best;\n  }"),
    "ready_any_parent": ("if (!done[dep_idx[e]]) { all_done = false; break; }",
                         "if (done[dep_idx[e]]) { all_done = true; break; } else all_done = false;"),
    "order_wf_desc": ("if (wf[a] != wf[b]) return wf[a] < wf[b];",
                      "if (wf[a] != wf[b]) return wf[a] > wf[b];"),
    "order_slack_desc": ("if (ka != kb) return ka < kb;", "if (ka != kb) return ka > kb;"),
    "lpt_shortest_first": ("return lpt ? -rem[v] : (srtf ? rem[v] : slack[v]);",
                           "return lpt ? rem[v] : (srtf ? rem[v] : slack[v]);"),
    "srtf_longest_first": ("return lpt ? -rem[v] : (srtf ? rem[v] : slack[v]);",
                           "return lpt ? -rem[v] : (srtf ? -rem[v] : slack[v]);"),
    "route_load_and_service_swapped": ("int64_t c = inst_load[i] + (est[v] * 1000) / inst_speed[i];",
                                       "int64_t c = est[v] + (inst_load[i] * 1000) / inst_speed[i];"),
    "route_penalty_without_loc_test": ("inst_speed[i];\n      if (loc[v] >= 0 && loc[v] != i) c += mig;",
                                       "inst_speed[i];\n      if (loc[v] >= 0) c += mig;"),
    "weighted_interval_off_by_one": ("if (r < int64_t(inst_weight[i])) pick = int32_t(i);",
                                     "if (r <= int64_t(inst_weight[i])) pick = int32_t(i);"),
    "weighted_one_sequence_for_all_types": ("int64_t r = next_seq[type[v]]++ % total;",
                                            "int64_t r = next_seq[0]++ % total;"),
    "weighted_pin_takes_a_number": ("if ((policy & kStateful) && loc[v] >= 0 && inst_type[loc[v]] == type[v]) continue;",
                                    "if ((policy & kStateful) && loc[v] >= 0 && inst_type[loc[v]] == type[v]) { next_seq[type[v]]++; continue; }"),
    "weighted_cost_without_penalty": ("(est[v] * 1000) / inst_speed[pick] +\n                ((loc[v] >= 0 && loc[v] != pick) ? mig : 0);",
                                      "(est[v] * 1000) / inst_speed[pick];"),
    "stateful_pays_penalty": ("cost[v] = inst_load[i] + (est[v] * 1000) / inst_speed[i];",
                              "cost[v] = inst_load[i] + (est[v] * 1000) / inst_speed[i] + mig;"),
    "greedy_no_load_update": ("        load[arg] += (est[v] * 1000) / inst_speed[arg];\n", ""),
    "greedy_adds_cost": ("load[arg] += (est[v] * 1000) / inst_speed[arg];", "load[arg] += best;"),
    "priority_low_first": ("return priority[wf[a]] > priority[wf[b]];",
                           "return priority[wf[a]] < priority[wf[b]];"),
    "stateful_any_type": ("if ((policy & kStateful) && loc[v] >= 0 && inst_type[loc[v]] == type[v]) {\n      const int32_t i",
                          "if ((policy & kStateful) && loc[v] >= 0) {\n      const int32_t i"),
    "max_with_first_successor_only": (
        "for (int64_t k = succ_off[v]; k < succ_off[v + 1]; ++k) best = std::max(best, rem[succ[k]]);",
        "if (succ_off[v] < succ_off[v + 1]) best = rem[succ[succ_off[v]]];"),
}


def _build_mutant(tmp_path, name):
    src = open(oracle.SRC).read()
    old, new = MUTATIONS[name]
    assert src.count(old) == 1, name
    path = tmp_path / f"{name}.cpp"
    path.write_text(src.replace(old, new))
    lib = tmp_path / f"lib{name}.so"
    subprocess.run(["g++", *oracle.CXXFLAGS, str(path), "-o", str(lib)], check=True)
    return str(lib)


def _pins_pass(lib_path):
    """Run the golden, brute-force, readiness and certificate pins with the
    given library swapped in; return True if all of them pass."""
    saved = oracle._lib
    lib = ctypes.CDLL(lib_path)
    lib.nalar_oracle_pass.restype = ctypes.c_int
    lib.nalar_oracle_pass.argtypes = [ctypes.c_int64] * 6 + [ctypes.c_void_p] * 17
    lib.nalar_oracle_pass_policy.restype = ctypes.c_int
    lib.nalar_oracle_pass_policy.argtypes = [ctypes.c_int64] * 6 + [ctypes.c_uint32] + [ctypes.c_void_p] * 19
    oracle._lib = lib
    try:
        for g in golden_names():
            p, exp = load_golden(g)
            r = oracle.run(p)
            if r.status != exp["status"][0] or r.order.tolist() != exp["order"] or \
               r.slack.tolist() != exp["slack"] or r.route.tolist() != exp["route"] or \
               r.cost.tolist() != exp["cost"] or r.rem.tolist() != exp["rem"]:
                return False
        for seed in range(40):
            p = wl.random_dag(seed, n_nodes=9, n_workflows=2, n_instances=4)
            r = oracle.run(p)
            if not np.array_equal(r.rem, brute_force_rem(p)):
                return False
            if set(r.order.tolist()) != push_replay_ready(p):
                return False
            keys = [(int(s), int(p.wf[v]), int(v)) for v, s in zip(r.order, r.slack)]
            if any(a >= b for a, b in zip(keys, keys[1:])):
                return False
            try:
                rem_certificate(p, r.rem)
                assert_routes_exhaustive(p, r)
                if seed % 4 == 0 and p.n_instances > 0:
                    q = wide_range(p, seed)
                    assert_routes_exhaustive(q, oracle.run(q))
            except AssertionError:
                return False
        for pin in (test_lpt_equals_srtf_when_deadlines_are_equal,
                    test_lpt_independent_futures_closed_form, test_stateful_routing_pins,
                    test_greedy_single_instance_prefix_sums,
                    test_greedy_identical_instances_round_robin):
            try:
                pin()
            except AssertionError:
                return False
        for pin in (test_priority_levels_partition_the_order, test_weighted_against_quota_walk):
            try:
                pin("tiny")
            except AssertionError:
                return False
        for pin in (test_srtf_independent_futures_closed_form, test_weighted_rules,
                    test_weighted_whole_periods_are_proportional):
            try:
                pin()
            except AssertionError:
                return False
        return True
    finally:
        oracle._lib = saved


def test_unmutated_oracle_passes_pins():
    assert _pins_pass(oracle.build())


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutant_is_caught(tmp_path, name):
    assert not _pins_pass(_build_mutant(tmp_path, name)), f"mutation {name} survived the pins"
