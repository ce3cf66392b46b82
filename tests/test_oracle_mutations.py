"""Plant plausible mistakes in copies of the oracle (on the CPU) and check that
the pins catch every one of them: a dropped term, a wrong sign, a wrong or
transposed index, a wrong order, an off-by-one offset, and the usual Adam slips
(no bias correction, eps inside the square root, the other eps placement, a
swapped beta).  Each mutant is compiled with gcc into a temporary directory."""
import os

import pytest

import oracle
import pins

SRC = open(oracle.SRC_PATH).read()

MUTANTS = {
    "gather_reversed_columns": ("W[id * D + j]", "W[id * D + (D - 1 - j)]", ["pin_gather"]),
    "coalesce_dropped_first_term": ("for (int64_t i = s; i < e; ++i) {", "for (int64_t i = s + 1; i < e; ++i) {",
                                    ["pin_coalesce_golden", "pin_coalesce_bruteforce"]),
    "coalesce_wrong_sign": ("acc[j] += g;", "acc[j] -= g;", ["pin_coalesce_golden", "pin_coalesce_bruteforce"]),
    "coalesce_index_by_id_not_token": ("c[i].t * D + j", "c[i].id * D + j",
                                       ["pin_coalesce_golden", "pin_coalesce_bruteforce"]),
    "coalesce_descending_ids": ("return x->id < y->id ? -1 : 1;", "return x->id < y->id ? 1 : -1;",
                                ["pin_coalesce_golden", "pin_coalesce_invariants"]),
    "coalesce_offsets_at_segment_end": ("seg_offsets[U] = (int32_t)s;", "seg_offsets[U] = (int32_t)e;",
                                        ["pin_coalesce_golden", "pin_coalesce_bruteforce"]),
    "pack_descending_inside_owner": ("int64_t pos = (int64_t)send_offsets[own[k]] + run[own[k]]++;",
                                     "int64_t pos = (int64_t)send_offsets[own[k] + 1] - 1 - run[own[k]]++;",
                                     ["pin_pack_golden", "pin_pack_invariants"]),
    "pack_owner_shifted": ("own[k] = row_owner[id];", "own[k] = (row_owner[id] + 1) % P;",
                           ["pin_pack_golden", "pin_pack_invariants"]),
    "split_inverted": ("is_prior[k] = bsearch(&key, nx, (size_t)T_next, sizeof(int32_t), orc_int32_cmp) != NULL;",
                       "is_prior[k] = bsearch(&key, nx, (size_t)T_next, sizeof(int32_t), orc_int32_cmp) == NULL;",
                       ["pin_split_golden", "pin_split_invariants"]),
    "split_drops_smallest_next_id": ("bsearch(&key, nx, (size_t)T_next,", "bsearch(&key, nx + 1, (size_t)(T_next > 0 ? T_next - 1 : 0),",
                                     ["pin_split_golden", "pin_split_invariants"]),
    "request_keeps_duplicates": ("if (k == 0 || u[k] != u[k - 1]) u[U++] = u[k];", "u[U++] = u[k];",
                                 ["pin_lookup_request_golden", "pin_lookup_request_invariants"]),
    "request_skipped_token_reads_row_0": ("        inverse[t] = -1;\n", "        inverse[t] = 0;\n",
                                          ["pin_lookup_request_golden", "pin_lookup_request_invariants"]),
    "request_groups_by_id_only": ("req_ids[req_offsets[p] + run[p]++] = u[k];", "req_ids[k] = u[k];",
                                  ["pin_lookup_request_golden", "pin_lookup_request_invariants"]),
    "request_inverse_local_to_owner": ("inverse[t] = hit != NULL ? (int32_t)(hit - req_ids) : -1;",
                                       "inverse[t] = hit != NULL ? (int32_t)(hit - blk) : -1;",
                                       ["pin_lookup_request_golden", "pin_lookup_request_invariants",
                                        "pin_lookup_request_serves_the_lookup"]),
    "column_split_rounds_up": ("return p * D / P;", "return (p * D + P - 1) / P;",
                               ["pin_column_golden", "pin_column_layout"]),
    "column_block_base_by_rows": ("blocks[C * a + r * w + j] = rows[r * D + a + j];",
                                  "blocks[R * a + r * w + j] = rows[r * D + a + j];",
                                  ["pin_column_golden", "pin_column_layout", "pin_column_roundtrip"]),
    "column_block_column_major": ("blocks[C * a + r * w + j] = rows[r * D + a + j];",
                                  "blocks[C * a + j * R + r] = rows[r * D + a + j];",
                                  ["pin_column_golden", "pin_column_layout", "pin_column_roundtrip"]),
    "column_join_ignores_row0": ("rows[r * D + a + j] = blocks[C * a + (row0 + r) * w + j];",
                                 "rows[r * D + a + j] = blocks[C * a + r * w + j];",
                                 ["pin_column_golden", "pin_column_roundtrip", "pin_column_forward"]),
    "column_lookup_token_for_id": ("ok ? shard[id * w + j] : 0.0f;", "ok ? shard[(t % V) * w + j] : 0.0f;",
                                   ["pin_column_golden", "pin_column_forward"]),
    "comm_alltoall_once": ("case 0: return 2.0 * (n - 1.0)", "case 0: return (n - 1.0)",
                           ["pin_comm_cost_golden", "pin_comm_cost_claims"]),
    "comm_alltoall_whole_gradient": ("(alpha * M / (n * B) + beta);", "(alpha * M / B + beta);",
                                     ["pin_comm_cost_golden", "pin_comm_cost_claims"]),
    "comm_ps_n_minus_1": ("case 2: return 2.0 * n *", "case 2: return 2.0 * (n - 1.0) *",
                          ["pin_comm_cost_golden", "pin_comm_cost_claims"]),
    "comm_allgather_n": ("case 3: return (n - 1.0)", "case 3: return n",
                         ["pin_comm_cost_golden", "pin_comm_cost_claims"]),
    "adam_no_bias_correction": ("double mhat = mm / bc1;", "double mhat = mm;",
                                ["pin_adam_golden", "pin_adam_closed_forms", "pin_adam_vs_torch_dense"]),
    "adam_eps_inside_sqrt": ("(sqrt(vhat) + eps)", "sqrt(vhat + eps)",
                             ["pin_adam_golden", "pin_adam_closed_forms", "pin_adam_vs_torch_dense"]),
    "adam_eps_on_uncorrected_v": ("lr * mhat / (sqrt(vhat) + eps)", "lr * sqrt(bc2) / bc1 * mm / (sqrt(vv) + eps)",
                                  ["pin_adam_closed_forms", "pin_adam_vs_torch_dense"]),
    "adam_swapped_beta": ("(1.0 - beta1) * g;", "(1.0 - beta2) * g;",
                          ["pin_adam_golden", "pin_adam_closed_forms", "pin_adam_vs_torch_dense"]),
    "adam_step_off_by_one": ("pow(beta1, (double)step)", "pow(beta1, (double)(step + 1))",
                             ["pin_adam_golden", "pin_adam_closed_forms", "pin_adam_vs_torch_dense"]),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_planted_mistake(name, tmp_path):
    find, repl, which = MUTANTS[name]
    assert SRC.count(find) == 1, f"mutation site not unique: {find!r}"
    lib = oracle.build_variant(SRC.replace(find, repl), os.path.join(str(tmp_path), f"lib_{name}.so"))
    caught = []
    try:
        oracle.use_library(lib)
        for pin in which:
            try:
                getattr(pins, pin)()
            except AssertionError:
                caught.append(pin)
    finally:
        oracle.use_library(None)
    assert caught, f"mutant {name} survived pins {which}"
