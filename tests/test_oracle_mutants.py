"""The pins are sensitive: plausible mistakes planted in a copy of the oracle
(compiled on the CPU into a temporary library) must each fail a pin test."""

import os
import subprocess

import pytest

import oracle
from tests import test_oracle_pins as pins

# (name, exact text in the oracle source, replacement, pin tests expected to fail)
MUTANTS = [
    ("self_not_in_mask", "for (int a = n; a >= 0; a = parent[node_off[b] + a])",
     "for (int a = parent[node_off[b] + n]; a >= 0; a = parent[node_off[b] + a])",
     ["test_random_trees_match_masked_sdpa"]),
    ("gqa_mapping", "int kv = h / group;", "int kv = h % n_kv;",
     ["test_gqa_equals_mha_with_repeated_kv"]),
    ("scale_dropped", "s[t] = scale * acc;", "s[t] = acc;",
     ["test_chain_tree_is_causal_attention"]),
    ("values_from_keys", "acc += s[t] * widen(V, dt,", "acc += s[t] * widen(K, dt,",
     ["test_single_node_is_decode_attention"]),
    ("tie_to_higher_id", "(va == vb && ia < ib)", "(va == vb && ia > ib)",
     ["test_topk_equals_stable_sort_with_ties", "test_greedy_acceptance_equals_brute_force"]),
    ("operand_reversed", "row[c] = widen(W, dt, iv * hidden + c);",
     "row[c] = widen(W, dt, iv * hidden + (hidden - 1 - c));",
     ["test_head_logits_equal_float64_matmul"]),
    ("rank_reversed", "* kmax + rank[n]];", "* kmax + (kmax - 1 - rank[n])];",
     ["test_tree_tokens_level_i_holds_head_i"]),
    ("threshold_max", "double thr = eps < delta", "double thr = eps > delta",
     ["test_typical_acceptance_equals_brute_force"]),
    ("entropy_sign", "hsum -= exp(lp) * lp;", "hsum += exp(lp) * lp;",
     ["test_typical_acceptance_equals_brute_force"]),
    ("no_move", "slab + (size_t)(L + pb[j]) * rb", "slab + (size_t)(L + j) * rb",
     ["test_compaction_moves_accepted_rows_only"]),
    ("pad_not_masked", "if (key_valid && t < L && !key_valid[rows[t]])", "if (key_valid && t < 0 && !key_valid[rows[t]])",
     ["test_padded_attention_equals_attention_without_pad_rows"]),
    ("pad_mask_on_tree_rows", "if (key_valid && t < L && !key_valid[rows[t]])", "if (key_valid && !key_valid[rows[t]])",
     ["test_padded_attention_equals_attention_without_pad_rows"]),
    ("resblock_no_residual", "out[((int64_t)i * B + b) * hidden + c] = x + acc / (1.0 + exp(-acc));",
     "out[((int64_t)i * B + b) * hidden + c] = acc / (1.0 + exp(-acc));",
     ["test_resblock_equals_torch_linear_silu"]),
    ("philox_weyl", "k1 += 0xBB67AE8584CAA73Bull;", "k1 += 0xBB67AE8584CAA73Aull;",
     ["test_philox_equals_numpy_stream"]),
    ("gumbel_sign", "g[i] = -log(-log(u));", "g[i] = log(-log(u));",
     ["test_sampled_token_follows_softmax", "test_gumbel_words_give_finite_standard_gumbel_values"]),
    ("gumbel_24_bits", "double u = ((double)(x[i] >> 41) + 0.5) / 8388608.0;",
     "double u = (double)(float)(((float)(x[i] >> 40) + 0.5f) * 0x1p-24f);",
     ["test_gumbel_words_give_finite_standard_gumbel_values"]),
    ("temperature_dropped", "double s = widen(logits, dt, row * vocab + v0 + j) * (double)inv_temp + g[j];",
     "double s = widen(logits, dt, row * vocab + v0 + j) + g[j];",
     ["test_sampled_token_follows_softmax"]),
    ("seq_len_off_by_one", "seq_len[b] = L + a + 1;", "seq_len[b] = L + a;",
     ["test_compaction_moves_accepted_rows_only"]),
]


def _call(name):
    fn = getattr(pins, name)
    marks = getattr(fn, "pytestmark", [])
    params = [m for m in marks if m.name == "parametrize"]
    if not params:
        fn()
        return
    argnames = [a.strip() for a in params[0].args[0].split(",")]
    for values in params[0].args[1]:
        values = values if isinstance(values, tuple) else (values,)
        fn(**dict(zip(argnames, values)))


@pytest.mark.parametrize("name,old,new,tests", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(tmp_path, name, old, new, tests):
    src = open(oracle.SRC).read()
    assert src.count(old) == 1, f"mutation anchor for {name} not unique"
    mut = tmp_path / "mut.c"
    mut.write_text(src.replace(old, new))
    so = tmp_path / "libmut.so"
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared", "-o", str(so),
                           str(mut), "-lm"])
    import ctypes
    saved = oracle._lib
    oracle._lib = ctypes.CDLL(str(so))
    try:
        caught = False
        for t in tests:
            try:
                _call(t)
            except AssertionError:
                caught = True
        assert caught, f"mutant {name} passed {tests}"
    finally:
        oracle._lib = saved
