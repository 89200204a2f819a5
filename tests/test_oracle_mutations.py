"""Mutation check of the oracle's pins: plant one plausible mistake at a time
in a copy of oracle/oracle.c (a flipped tie-break, a dropped term, a floor for
a ceiling, a skipped pass, a wrong index), build it, and require that at
least one pin or invariant check fails.  Runs on the CPU only."""
import os
import subprocess
import sys

import pytest

import test_oracle_pins as pins

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                   "oracle", "oracle.c")

# Not listed: dropping the probe's "expert already on t" guard.  After a
# transfer of e to t either t's slack is spent (delta = slack) or e's loop
# ends (delta = excess or cap), so the guard never decides a target and the
# mutant is equivalent (the oracle asserts this as its lemma flag).
MUTATIONS = {
    "argmax_tie_to_higher_rank": ("if (best < 0 || slk[t] > slk[best]) best = t;",
                                  "if (best < 0 || slk[t] >= slk[best]) best = t;"),
    "delta_ignores_cap": ("int64_t delta = min64(min64(exc[r], slk[best]), cap);",
                          "int64_t delta = min64(exc[r], slk[best]);"),
    "u_min_inclusive": ("if (delta < g->u_min) break;",
                        "if (delta <= g->u_min) break;"),
    "mid_rounds_up": ("int64_t tau = (lo + hi) / 2;",
                      "int64_t tau = (lo + hi + 1) / 2;"),
    "tau_lo_floor": ("*lo = (g->beta_num * m + g->beta_den - 1) / g->beta_den;",
                     "*lo = g->beta_num * m / g->beta_den;"),
    "mean_floor": ("int64_t m = (c->L + g->R - 1) / g->R;",
                   "int64_t m = c->L / g->R;"),
    "no_locality": ("int64_t q = locality ? min64(lamhat[t], u) : 0;",
                    "int64_t q = 0;"),
    "remainder_tie_to_later_host": (
        "if (!taken[i] && (best < 0 || rem[i] > rem[best])) best = i;",
        "if (!taken[i] && (best < 0 || rem[i] >= rem[best])) best = i;"),
    "order_ascending": ("if (x->key != y->key) return x->key > y->key ? -1 : 1;",
                        "if (x->key != y->key) return x->key < y->key ? -1 : 1;"),
    "order_ties_to_higher_id": ("return x->id < y->id ? -1 : (x->id > y->id);",
                                "return x->id > y->id ? -1 : (x->id < y->id);"),
    "replica_pslot_without_main_offset": ("host_pslot[j] = nm + s;",
                                          "host_pslot[j] = s;"),
    "lookup_inclusive": ("if (j < C + qi) {", "if (j <= C + qi) {"),
    "pack_slot_major": (
        "  for (int32_t t = 0; t < R; t++)\n    for (int32_t s = 0; s < NS; s++) {\n      int32_t e = slot_expert[(int64_t)t * NS + s];\n      if (e >= 0 && home(g, e) == rank) {\n        memcpy",
        "  for (int32_t s = 0; s < NS; s++)\n    for (int32_t t = 0; t < R; t++) {\n      int32_t e = slot_expert[(int64_t)t * NS + s];\n      if (e >= 0 && home(g, e) == rank) {\n        memcpy"),
    "proportional_split_on_full_quota": ("uhat[i] = u - q; /* residual quota */",
                                         "uhat[i] = u; /* residual quota */"),
    "residual_not_updated": ("        uhat[i] -= qv[i];\n", "\n"),
    "home_keeps_nothing_back": ("Ut[(int64_t)e * R + home(g, e)] -= delta;",
                                "Ut[(int64_t)e * R + home(g, e)] -= 0;"),
    "relay_threshold_inclusive": (
        "if (host_ptr[e + 1] - host_ptr[e] - 1 > threshold) hot[nhot++] = e;",
        "if (host_ptr[e + 1] - host_ptr[e] - 1 >= threshold) hot[nhot++] = e;"),
    "relay_frontier_floor": ("return f > n * n + n ? n + 1 : n;", "return n;"),
    "relay_hot_order_ascending": ("if (fp > fe || (fp == fe && p < e)) break;",
                                  "if (fp < fe || (fp == fe && p < e)) break;"),
    "relay_picks_largest_volume": (
        "if (best < 0 || vol[t] < vol[best] || (vol[t] == vol[best] && t < best)) best = t;",
        "if (best < 0 || vol[t] > vol[best] || (vol[t] == vol[best] && t < best)) best = t;"),
    "relay_leaf_tie_to_larger_rank": (
        "if (best < 0 || vol[u] + 1 < vol[best] + 1 || (vol[u] == vol[best] && u < best)) best = u;",
        "if (best < 0 || vol[u] + 1 <= vol[best] + 1) best = u;"),
    "relay_leaf_volume_not_counted": ("      vol[best] += 1;\n      slot_src", "      slot_src"),
    "relay_source_not_updated": ("vol[home(g, e)] -= f - n;", "vol[home(g, e)] -= 0;"),
    "pack_relay_reads_main_blob": ("src = relay_src + (int64_t)s2 * W;", "src = w_main;"),
    "combine_k_descending": ("      for (int32_t kk = 0; kk < k; kk++) {\n        int32_t row = row_of_slot[t * k + kk];",
                             "      for (int32_t kk = k - 1; kk >= 0; kk--) {\n        int32_t row = row_of_slot[t * k + kk];"),
    "combine_ignores_gate": ("volatile float prod = gate[t * k + kk] * bf16_to_f32(",
                             "volatile float prod = bf16_to_f32("),
    "bf16_ties_away_from_zero": ("if (dropped > 0x8000u || (dropped == 0x8000u && (kept & 1u))) kept += 1;",
                                 "if (dropped >= 0x8000u) kept += 1;"),
    "bf16_truncates": ("if (dropped > 0x8000u || (dropped == 0x8000u && (kept & 1u))) kept += 1;",
                       "(void)dropped;"),
    "combine_accumulates_in_double": ("      volatile float acc = 0.0f; /* volatile",
                                      "      volatile double acc = 0.0f; /* volatile"),
    "grad_reduce_keeps_replicas": ("        rg[i] = 0.0f;\n", "\n"),
    "count_skips_expert_zero": ("      if (e == -1) continue;\n      if (e < -1 || e >= E) { status = ORC_EDATA; continue; }\n      c[e] += 1;",
                                "      if (e <= 0) continue;\n      if (e < -1 || e >= E) { status = ORC_EDATA; continue; }\n      c[e] += 1;"),
    "probe_slack_not_consumed": ("        slk[best] -= delta;\n", "\n"),
    "probe_excess_not_consumed": ("        exc[r] -= delta;\n", "\n"),
    "bisect_keeps_failed_tau": ("      lo = tau + 1;", "      lo = tau;"),
    "bisect_forgets_best": ("      if (U) memcpy(U, Ut, sizeof(int64_t) * (size_t)g->E * g->R);\n",
                            "\n"),
    "dispatch_copies_next_token": ("memcpy(send + (int64_t)row_of_slot[i] * H, x + (i / k) * H,",
                                   "memcpy(send + (int64_t)row_of_slot[i] * H, x + ((i / k + 1) % T) * H,"),
    "dispatch_tail_not_zeroed": ("    if (V > v_valid)\n      memset(", "    if (0)\n      memset("),
    "block_off_starts_at_first_block_size": ("  block_off[0] = 0;\n  for (int64_t b = 0; b < (int64_t)R * S; b++) block_off[b + 1]",
                                             "  block_off[0] = cnt[0];\n  for (int64_t b = 0; b < (int64_t)R * S; b++) block_off[b + 1]"),
    "x_slots_fill_from_the_end": ("        slots[(int64_t)best * NS + used[best]] = e;",
                                  "        slots[(int64_t)best * NS + (NS - 1 - used[best])] = e;"),
    "hosts_in_descending_rank_order": ("    for (int32_t t = 0; t < R; t++)\n      for (int32_t s = 0; s < NS; s++)\n        if (X[(int64_t)t * NS + s] == e) {",
                                       "    for (int32_t t = R - 1; t >= 0; t--)\n      for (int32_t s = 0; s < NS; s++)\n        if (X[(int64_t)t * NS + s] == e) {"),
    "residual_sources_descending": ("    for (int32_t r = 0; r < R; r++) {\n      if (lamhat[r] == 0) continue;",
                                    "    for (int32_t r = R - 1; r >= 0; r--) {\n      if (lamhat[r] == 0) continue;"),
    "pack_counts_other_ranks_experts": ("    dest_off[t] = n;\n    for (int32_t s = 0; s < NS; s++) {\n      int32_t e = slot_expert[(int64_t)t * NS + s];\n      if (e >= 0 && home(g, e) == rank) n++;\n    }\n  }\n  dest_off[R] = n;\n  *n_out = n;\n  if (n > cap) return ORC_ENOSPC;\n  if (n > 0 && !staging) return ORC_EINVAL;",
                                        "    dest_off[t] = n;\n    for (int32_t s = 0; s < NS; s++) {\n      int32_t e = slot_expert[(int64_t)t * NS + s];\n      if (e >= 0) n++;\n    }\n  }\n  dest_off[R] = n;\n  *n_out = n;\n  if (n > cap) return ORC_ENOSPC;\n  if (n > 0 && !staging) return ORC_EINVAL;"),
    "grad_reduce_slot_major": (
        "  n = 0;\n  for (int32_t t = 0; t < R; t++)\n    for (int32_t s = 0; s < NS; s++) {\n      int32_t e = slot_expert[(int64_t)t * NS + s];\n      if (e < 0 || home(g, e) != rank) continue;\n      float *mg",
        "  n = 0;\n  for (int32_t s = 0; s < NS; s++)\n    for (int32_t t = 0; t < R; t++) {\n      int32_t e = slot_expert[(int64_t)t * NS + s];\n      if (e < 0 || home(g, e) != rank) continue;\n      float *mg"),
}


RUNNER = os.path.join(os.path.dirname(os.path.abspath(__file__)),
                      "mutation_runner.py")


@pytest.fixture(scope="module")
def bruteforce(tmp_path_factory):
    return pins.build_bruteforce(tmp_path_factory.mktemp("bfm"))


def _run(lib_path, bf, timeout=120):
    """Exit code of the pin harness on one build; a hang counts as a failure
    (returned as 124)."""
    try:
        return subprocess.run([sys.executable, RUNNER, lib_path, bf],
                              capture_output=True, text=True,
                              timeout=timeout).returncode
    except subprocess.TimeoutExpired:
        return 124


def test_unmutated_oracle_passes_the_harness(orc, bruteforce):
    assert _run(orc._LIB, bruteforce) == 0


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutation_is_caught(bruteforce, tmp_path, name):
    old, new = MUTATIONS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation anchor not unique/found: {name}"
    mdir = tmp_path / name
    mdir.mkdir()
    (mdir / "oracle.c").write_text(src.replace(old, new))
    (mdir / "oracle.h").write_text(open(SRC[:-2] + ".h").read())
    so = str(mdir / "libmut.so")
    subprocess.run(["gcc", "-O1", "-std=c11", "-ffp-contract=off", "-fPIC", "-shared", "-o", so,
                    str(mdir / "oracle.c")], check=True)
    # exit 3: a pin failed; a crash or a hang is also a detection
    assert _run(so, bruteforce, timeout=30) != 0, f"no pin detects {name}"
