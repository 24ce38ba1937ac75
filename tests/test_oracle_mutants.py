"""Planted mistakes in the oracle must be caught by its pins.

Each case copies the oracle source, plants one plausible mistake (a dropped
term, a wrong sign or index, a swapped operand, another reading of the
paper), builds it with gcc on the CPU, and runs every pin against it: at
least one pin must fail.
"""
import os
import shutil
import tempfile

import pytest

import oracle
import oracle_pins
from oracle import build as obuild

MUTANTS = {
    # step 1: exclusive instead of inclusive running sum
    "cdf_off_by_one": ("running += counts[k];\n        cdf[k + 1] = (double)running / (double)total;",
                       "cdf[k + 1] = (double)running / (double)total;\n        running += counts[k];"),
    # step 3: the batch takes the fastest member's CDF (min instead of max)
    "cdf_product_to_max": ("G[k] *= Fn[k];", "G[k] = G[k] > Fn[k] ? G[k] : Fn[k];"),
    # step 3: identical members only (ignores class of later members)
    "first_class_only": ("(size_t)cls[n - 1]) * row;", "(size_t)cls[0]) * row;"),
    # step 4: dropped half of the trapezoid
    "el_dropped_term": ("el += 1.0 - 0.5 * (G[k] + G[k + 1]);", "el += 1.0 - G[k + 1];"),
    # step 5: interpolation weights swapped
    "p_swapped_weights": ("return (1.0 - theta) * G[k] + theta * G[k + 1];",
                          "return theta * G[k] + (1.0 - theta) * G[k + 1];"),
    # step 5: dead requests treated as finishing
    "p_dead_finishes": ("if (!(tau > 0.0))\n        return 0.0;",
                        "if (!(tau > 0.0))\n        return G[n_bins];"),
    # step 5: requests beyond the grid treated as missing
    "p_beyond_misses": ("if (u >= (double)n_bins)\n        return G[n_bins];",
                        "if (u >= (double)n_bins)\n        return 0.0;"),
    # step 7: wrong sign in the delay exponent
    "eq2_sign": ("exp(-b * (tau - l2)) - exp(-b * (tau - l1))",
                 "exp(b * (tau - l2)) - exp(b * (tau - l1))"),
    # step 7: case 2 measured from the upper edge
    "eq2_case2_edge": ("acc += h / b * (1.0 - exp(-b * (tau - l1)));",
                       "acc += h / b * (1.0 - exp(-b * (tau - l2)));"),
    # step 7: literal "frequency" reading (mass, not density)
    "eq2_mass_not_density": ("double h = mass[i] / w;", "double h = mass[i];"),
    # step 7: case 2 dropped
    "eq2_case2_dropped": ("else if (tau > l1)", "else if (tau > l1 + 1e300)"),
    # step 7: bin masses from the wrong neighbour
    "mass_index": ("mass[k] = G[k + 1] - G[k];", "mass[k] = G[k + 1] - G[k > 0 ? k - 1 : 0];"),
    # step 6/7: priority not divided by E[L_B]
    "priority_not_normalised": ("priority_times_latency(mass, K, w, tau, b) / el;",
                                "priority_times_latency(mass, K, w, tau, b);"),
    # step 8: exact ties to the larger batch size
    "select_tie_bs": ("(s == bt->score && n > bt->n)", "(s == bt->score && n >= bt->n)"),
    # step 8: no-batch rule dropped
    "select_nonpositive": ("if (bt->have && bt->score > 0.0) {", "if (bt->have) {"),
    # step 8: over-long prefixes allowed
    "select_rect_mask": ("if (n <= bs) {", "if (1) {"),
    # Algorithm 1: the request's batch holds s mix members besides it
    "iter_mix_power": ("G[k] = Fr[k] * pow(mix[k], s - 1);", "G[k] = Fr[k] * pow(mix[k], s);"),
    # Algorithm 1: model-wide E[L] of s - 1 mix members
    "iter_el_power": ("pow(mix[k], s) + pow(mix[k + 1], s)",
                      "pow(mix[k], s - 1) + pow(mix[k + 1], s - 1)"),
    # Algorithm 1: the class mix ignores the weights
    "iter_weights_ignored": ("double pc = weights ? weights[c] / wsum : 1.0 / (double)C;",
                             "double pc = 1.0 / (double)C;"),
    # Algorithm 1: a request is kept at every batch size
    "iter_drop_never": ("if (finish_probability(Fr, K, w, tau) > 0.0) {",
                        "if (finish_probability(Fr, K, w, tau) >= 0.0) {"),
    # Algorithm 1: candidate order ascending in D_{Q_s}
    "iter_cand_order": ("if (d_new > d_old || (d_new == d_old && batch_sizes[bi] > batch_sizes[cand]))",
                        "if (d_new < d_old || (d_new == d_old && batch_sizes[bi] > batch_sizes[cand]))"),
    # miss costs ignored in the score
    "cost_ignored": ("s += (cost ? cost[m - 1] : 1.0) * p;", "s += p;"),
    # App. B: cumulative costs used as increments
    "steps_cumulative": ("pr += (step_cost[j] - below) * priority_times_latency(dG, K, w, tau_j, b);",
                         "pr += step_cost[j] * priority_times_latency(dG, K, w, tau_j, b);"),
    # App. B: the drop phase looks at the first step
    "steps_drop_first": ("double last = step_off ? step_deadline_ms[step_off[r + 1] - 1] : deadline_ms[r];\n        double tau = last - now_ms;",
                         "double last = deadline_ms[r];\n        double tau = last - now_ms;"),
    # Eq. (3): the overhead c0 ignored in the finish probability
    "affine_p_no_c0": ("finish_probability(G, K, ws, tau - c0_ms)", "finish_probability(G, K, ws, tau)"),
    # Eq. (3): the priority measured from the batch start, not after c0
    "affine_priority_no_c0": ("priority_times_latency(hist, K, ws, tau - c0_ms, b)",
                              "priority_times_latency(hist, K, ws, tau, b)"),
    # Eq. (9): the L_B grid not stretched by the batch size
    "affine_width_no_k": ("const double ws = c1 * (double)batch_sizes[bi] * w;",
                          "const double ws = c1 * w;"),
    # Eq. (5): c0 dropped from E[L_B]
    "affine_el_no_c0": ("const double el = c0_ms + c1 * (double)batch_sizes[bi] * ex;",
                        "const double el = c1 * (double)batch_sizes[bi] * ex;"),
    # Eq. (5): E[L_B] without the factor k
    "affine_el_no_k": ("const double el = c0_ms + c1 * (double)batch_sizes[bi] * ex;",
                       "const double el = c0_ms + c1 * ex;"),
    # profiler: beyond-grid samples dropped instead of counted in the last bin
    "accumulate_clip": ("int32_t k = u >= (double)(n_bins - 1) ? n_bins - 1 : (int32_t)u;",
                        "if (u >= (double)n_bins) { ++rejected; continue; }\n        int32_t k = (int32_t)u;"),
    # profiler: bin by rounding instead of flooring
    "accumulate_round": ("double u = floor(lat / bin_width_ms[q]);", "double u = floor(lat / bin_width_ms[q] + 0.5);"),
    # Algorithm 1: PopBatch takes the lowest priorities
    "iter_pop_lowest": ("if (si > sb || (si == sb && order[i] < order[best]))",
                        "if (si < sb || (si == sb && order[i] < order[best]))"),
}


@pytest.fixture(scope="module")
def src_text():
    with open(obuild.SRC) as f:
        return f.read()


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, src_text):
    old, new = MUTANTS[name]
    assert src_text.count(old) == 1, f"mutation anchor for {name} not unique/found"
    d = tempfile.mkdtemp(prefix="oracle_mut_")
    try:
        src = os.path.join(d, "mut.c")
        with open(src, "w") as f:
            f.write(src_text.replace(old, new))
        so = obuild.compile_oracle(src, os.path.join(d, f"lib_{name}.so"), extra=["-w"])
        L = oracle.lib(so)
        failed = []
        for pin in oracle_pins.PINS:
            try:
                pin(L)
            except (AssertionError, oracle.OracleError):
                failed.append(pin.__name__)
        assert failed, f"no pin caught mutant {name}"
    finally:
        shutil.rmtree(d, ignore_errors=True)
