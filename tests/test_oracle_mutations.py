"""Planted mistakes in the oracle (on the CPU): each must fail at least one pin.

Every mutant is a copy of oracle.c with one plausible slip (a dropped term,
a wrong sign, a swapped operand or index, a reversed tie-break, ...),
compiled to a temporary library.  The pins in oracle_pins.py are the
evidence that the oracle itself is right; this test shows they are strong
enough to notice such slips.
"""
import ctypes
import os

import pytest

import oracle
import oracle_pins

MUTANTS = {
    "dot_drops_last_term": ("for (int32_t t = 0; t < d; ++t) acc +=", "for (int32_t t = 0; t < d - 1; ++t) acc +="),
    "dot_wrong_operand_row": ("decode(b, dtype, brow + t)", "decode(b, dtype, qrow + t)"),
    "bf16_decode_shift": ("[i] << 16;", "[i] << 15;"),
    "softmax_sign": ("sum += exp(scale * c[t].s - mx);", "sum += exp(mx - scale * c[t].s);"),
    "lse_drops_max": ("return mx + log(sum);", "return log(sum);"),
    "prob_drops_scale": ("prob_out[i * k + r] = exp(scale * c[r].s - lse);",
                         "prob_out[i * k + r] = exp(c[r].s - lse);"),
    "tie_break_reversed": ("return (a->j < b->j) ? -1 : (a->j > b->j);", "return (a->j > b->j) ? -1 : (a->j < b->j);"),
    "selects_smallest": ("if (a->s > b->s) return -1;\n  if (a->s < b->s) return 1;",
                         "if (a->s < b->s) return -1;\n  if (a->s > b->s) return 1;"),
    "self_not_excluded": ("if (j == self) continue;", "if (j == self && 0) continue;"),
    "time_order_descending": ("while (p > g0 && out[p - 1] > v)", "while (p > g0 && out[p - 1] < v)"),
    "gather_ignores_page": ("int64_t page = table[(int64_t)c * ppc + p];", "int64_t page = table[(int64_t)c * ppc];"),
    "splitmix_wrong_shift": ("z = (z ^ (z >> 27))", "z = (z ^ (z >> 28))"),
    "payload_page_index": ("(uint64_t)((chunk * ppc + page) * wpp)", "(uint64_t)((chunk + page) * wpp)"),
    "append_off_by_one": ("(int32_t)(next_free + r * ppc + p)", "(int32_t)(next_free + r * ppc + p + 1)"),
    "scoped_ignores_tombstones": ("if (j == self || !row_live[j] || row_ns[j] != key_ns[i]) continue;",
                                  "if (j == self || row_ns[j] != key_ns[i]) continue;"),
    "scoped_ignores_namespace": ("if (j == self || !row_live[j] || row_ns[j] != key_ns[i]) continue;",
                                 "if (j == self || !row_live[j]) continue;"),
    "scoped_pads_with_zero_id": ("idx_out[i * k + r] = have ? (int32_t)c[r].j : -1;",
                                 "idx_out[i * k + r] = have ? (int32_t)c[r].j : 0;"),
    "budget_skips_and_continues": ("if (total + tok_len[c] > budget) break;",
                                   "if (total + tok_len[c] > budget) continue;"),
    "budget_strict": ("if (total + tok_len[c] > budget) break;", "if (total + tok_len[c] >= budget) break;"),
    "budget_rank_order_kept": ("oracle_time_order(ranked, nk, nk > 0 ? nk : 1, kept);",
                               "memcpy(kept, ranked, (size_t)nk * sizeof(int32_t));"),
    "budget_token_page_swapped": ("table[(int64_t)c * ppc + t / tpp]", "table[(int64_t)c * ppc + t % ppc]"),
    "compact_phi_counts_live": ("const double phi = (double)(written - live[b]) / (double)P;",
                                "const double phi = (double)(live[b]) / (double)P;"),
    "compact_strict_theta": ("phi >= theta;", "phi > theta;"),
    "compact_partial_block": ("cand[b] = ((b + 1) * P <= next_free) && phi >= theta;", "cand[b] = phi >= theta;"),
    "compact_mixes_namespaces": ("if (pos > start) pos = start + ((pos - start + P - 1) / P) * P;", "(void)start;"),
    "compact_pages_reversed": ("for (int32_t pp = 0; pp < ppc; ++pp) {", "for (int32_t pp = ppc - 1; pp >= 0; --pp) {"),
    "compact_dir_not_updated": ("          *entry = (int32_t)pos;\n", ""),
    "colocate_strict_tau": ("if ((double)scores[i * k + r] >= (double)tau)", "if ((double)scores[i * k + r] > (double)tau)"),
    "colocate_ignores_min_group": ("if (g < min_group) continue;", "(void)0;"),
    "colocate_moves_twice": ("if (!done[grp[a]]) {", "if (1) {"),
    "colocate_rank_order": ("oracle_time_order(grp, nk, nk, ord);", "memcpy(ord, grp, (size_t)nk * sizeof(int32_t));"),
    "colocate_dir_not_updated": ("*entry = (int32_t)pos; /* UpdateDir; the old copy is now invalid */", "(void)0;"),
    "budget_no_zero_tail": ("memset(dst + row * row_bytes, 0, (size_t)((budget - row) * row_bytes));",
                            "(void)0;"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(tmp_path, name):
    before, after = MUTANTS[name]
    src = open(os.path.join(os.path.dirname(oracle.__file__), "oracle.c")).read()
    assert src.count(before) == 1, f"mutation site for {name} not found exactly once"
    mpath = tmp_path / "mutant.c"
    mpath.write_text(src.replace(before, after))
    so = oracle.build(force=True, src=str(mpath), out=str(tmp_path / "libmutant.so"))
    L = oracle._bind(ctypes.CDLL(so))
    caught = []
    for pin in oracle_pins.PINS:
        try:
            pin(L)
        except (AssertionError, ValueError):
            caught.append(pin.__name__)
    assert caught, f"no pin notices mutant {name}"
