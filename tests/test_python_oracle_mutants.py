"""The pins of the Python oracles (budget and tree construction, padded
batching, the decode loop) are sensitive: a plausible mistake planted in a
copy of an oracle module's source must make at least one of its pins fail."""

import os
import sys
import types

import pytest

import oracle
from tests import test_budget_oracle as budget_pins
from tests import test_decode_oracle as decode_pins
from tests import test_oracle_pins as pins

HERE = os.path.dirname(os.path.abspath(oracle.__file__))


def _mutant(modname, old, new):
    path = os.path.join(HERE, modname + ".py")
    src = open(path).read()
    assert src.count(old) == 1, f"mutation anchor not unique in {modname}: {old!r}"
    mod = types.ModuleType(f"oracle.{modname}")
    mod.__file__ = path
    mod.__package__ = "oracle"
    exec(compile(src.replace(old, new), path, "exec"), mod.__dict__)
    return mod


def _fails(fn, *args):
    # only a failed check counts: a mutant that crashes a pin would hide a
    # badly planted mutation
    try:
        fn(*args)
    except AssertionError:
        return True
    return False


def _param_cases(fn):
    marks = [m for m in getattr(fn, "pytestmark", []) if m.name == "parametrize"]
    if not marks:
        return [()]
    return [v if isinstance(v, tuple) else (v,) for v in marks[0].args[1]]


BUDGET = [
    ("eq3_drops_acceptance_term", "+ batch * seqs * levels * levels * vocab", "",
     ["test_r1_buffer_model_reproduces_the_paper_numbers"]),
    ("eq1_without_head_dim", "return 2 * layers * batch * n_kv * head_dim * tokens * elem_bytes",
     "return 2 * layers * batch * n_kv * tokens * elem_bytes", ["test_r2_kv_model_with_head_dim"]),
    ("eq2_one_level_short", "for _ in range(levels + 1):", "for _ in range(levels):",
     ["test_r3_full_tree_closed_form"]),
    ("builder_depth_first", "for p in sorted(paths, key=lambda q: (len(q), q)):",
     "for p in sorted(paths, key=lambda q: q):", ["test_builder_feasibility_matches_brute_force"]),
    ("pruning_keeps_rightmost", "for n in range(len(parent)):\n            if depth[n] == d",
     "for n in reversed(range(len(parent))):\n            if depth[n] == d", ["test_pruning_right_to_left"]),
    ("plan_skips_fewer_heads", "for h in range(default_heads, 1, -1):", "for h in range(default_heads, 2, -1):",
     ["test_budget_plan_boundaries"]),
    ("tree_size_ignores_budget", "return [max(0, min(default_nodes, c - l)) for l, c in zip(seq_len, seq_cap)]",
     "return [default_nodes for l, c in zip(seq_len, seq_cap)]", ["test_tree_sizes_from_slab_capacity"]),
]


@pytest.mark.parametrize("name,old,new,tests", BUDGET, ids=[m[0] for m in BUDGET])
def test_budget_mutant_is_caught(monkeypatch, name, old, new, tests):
    mut = _mutant("budget", old, new)
    monkeypatch.setattr(budget_pins, "ob", mut)
    caught = [t for t in tests if any(_fails(getattr(budget_pins, t), *c) for c in _param_cases(getattr(budget_pins, t)))]
    assert caught, f"mutant {name} passed every pin"


PADDED = [
    ("no_padding", "T = int(tau.max()) if len(tau) else 0", "T = 0", ["test_fig8_padding_of_accepted_tokens"]),
    ("positions_count_pads", "new_pos = (np.asarray(pos, dtype=np.int64) + tau).astype(np.int32)",
     "new_pos = (np.asarray(pos, dtype=np.int64) + T).astype(np.int32)", ["test_fig8_padding_of_accepted_tokens"]),
    ("pads_flagged_valid", "key_valid[first + j] = 1 if j < tau[b] else 0", "key_valid[first + j] = 1",
     ["test_fig8_padding_of_accepted_tokens", "test_padded_steps_keep_the_tokens_of_compaction"]),
]


@pytest.mark.parametrize("name,old,new,tests", PADDED, ids=[m[0] for m in PADDED])
def test_padded_mutant_is_caught(monkeypatch, name, old, new, tests):
    mut = _mutant("padded", old, new)
    monkeypatch.setitem(sys.modules, "oracle.padded", mut)
    monkeypatch.setattr(oracle, "padded", mut, raising=False)
    caught = [t for t in tests if _fails(getattr(pins, t))]
    assert caught, f"mutant {name} passed every pin"


DECODE = [
    ("root_not_chained", "root[seqs] = nxt", "pass", ["test_decode_loop_bookkeeping"]),
    ("lengths_not_advanced", "lens[seqs] = new_len", "pass", ["test_decode_loop_bookkeeping"]),
    ("sampling_ignored", "        if setup.temperature is not None:\n",
     "        if False:\n", ["test_sampled_tokens_differ_from_greedy_and_follow_the_seed"]),
    ("typical_ignored", "        if setup.typical is not None:\n", "        if False:\n",
     ["test_typical_with_vanishing_thresholds_accepts_the_deepest_nodes"]),
]


@pytest.mark.parametrize("name,old,new,tests", DECODE, ids=[m[0] for m in DECODE])
def test_decode_mutant_is_caught(monkeypatch, name, old, new, tests):
    mut = _mutant("decode", old, new)
    monkeypatch.setattr(decode_pins, "decode", mut)
    caught = [t for t in tests if any(_fails(getattr(decode_pins, t), *c) for c in _param_cases(getattr(decode_pins, t)))]
    assert caught, f"mutant {name} passed every pin"


def test_unmutated_modules_pass(monkeypatch):
    # the loader itself changes nothing: an identity "mutation" passes the pins
    monkeypatch.setattr(budget_pins, "ob", _mutant("budget", "def kv_bytes(", "def kv_bytes("))
    for t in ("test_r1_buffer_model_reproduces_the_paper_numbers", "test_r2_kv_model_with_head_dim",
              "test_budget_plan_boundaries"):
        assert not _fails(getattr(budget_pins, t)), t
    monkeypatch.setattr(decode_pins, "decode", _mutant("decode", "def run(", "def run("))
    assert not _fails(decode_pins.test_sampled_tokens_differ_from_greedy_and_follow_the_seed)
