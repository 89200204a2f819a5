"""Runs the oracle pins against one build of oracle.c (used by
test_oracle_mutations in a child process).  Exit 0: every pin passed;
exit 3: some pin failed."""
import os
import sys

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

import gen  # noqa: E402
import oracle  # noqa: E402
import test_oracle_invariants as inv  # noqa: E402
import test_oracle_pins as pins  # noqa: E402
import test_oracle_combine_reduce as cr  # noqa: E402
import test_oracle_relay as relay  # noqa: E402


def main(lib_path, bf_exe):
    oracle.use_library(lib_path)
    orc = oracle
    checks = [
        lambda: [pins.test_worked_example_plan(orc, n) for n in
                 ("W0_single_hot_expert.json", "W1_nonmonotone_bisection.json",
                  "W2_proportional_split.json", "W4_two_slots_dispatch_pack.json",
                  "W5_visit_order.json", "W7_source_order.json")],
        lambda: pins.test_w6_pack_order(orc),
        lambda: pins.test_w1_feasibility_is_not_monotone(orc),
        lambda: pins.test_w3_rounding_keeps_both_margins(orc),
        lambda: pins.test_w4_dispatch_and_pack(orc),
        lambda: pins.test_apportion_matches_closest_vector_search(orc),
        lambda: pins.test_s1_no_slots_is_stable_counting_sort(orc),
        lambda: pins.test_s2_balanced_load_needs_no_probe(orc),
        lambda: [pins.test_s3_single_hot_expert_closed_form(orc, R) for R in (2, 5)],
        lambda: pins.test_bruteforce_small_random_groups(orc, bf_exe),
        lambda: [inv.test_fuzz_case(orc, s) for s in range(40)],
        lambda: relay.test_figure_nine_replicas_three_relays(),
        lambda: [relay.test_single_hot_expert_closed_form(f, n)
                 for f, n in sorted(relay.FRONTIER.items())],
        lambda: [relay.test_at_most_four_replicas_no_relay(f) for f in (1, 4)],
        lambda: relay.test_relays_avoid_busy_senders(),
        lambda: relay.test_second_hot_expert_sees_first_ones_volumes(),
        lambda: relay.test_larger_fanout_goes_first(),
        lambda: relay.test_pack_relay_stages_for_the_slots_a_rank_sends(),
        lambda: cr.test_combine_unit_weight_k1_is_a_copy(),
        lambda: [cr.test_combine_rounds_to_nearest_even(gt, w) for gt, w in
                 [(1 + 2 ** -8, 0x3F80), (1 + 3 * 2 ** -8, 0x3F82), (1 + 2 ** -8 + 2 ** -20, 0x3F81)]],
        lambda: [cr.test_combine_sums_in_fp32_in_k_order(o, w) for o, w in
                 [((2.0 ** 25, 1.0, -2.0 ** 25), 0), ((2.0 ** 25, -2.0 ** 25, 1.0), 0x3F80)]],
        lambda: [cr.test_combine_within_error_bound_of_the_fp64_definition(s, k) for s, k in ((0, 8), (1, 2))],
        lambda: cr.test_grad_reduce_integer_sums_are_exact(),
        lambda: cr.test_grad_reduce_fp32_sequential_from_the_main_value(),
        lambda: cr.test_grad_reduce_follows_staging_order(),
        lambda: cr.test_grad_reduce_entries_map_to_experts_in_staging_order(),
        lambda: cr.test_grad_reduce_within_error_bound_of_the_fp64_sum(0),
    ]
    for i, chk in enumerate(checks):
        try:
            chk()
        except Exception as ex:  # a failed pin
            print(f"caught by check {i}: {type(ex).__name__}: {str(ex)[:120]}")
            return 3
    return 0


if __name__ == "__main__":
    sys.exit(main(sys.argv[1], sys.argv[2]))
