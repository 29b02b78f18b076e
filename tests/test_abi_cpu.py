"""The C-ABI library loads, exports what include/specmemo.h declares, and
rejects bad arguments on the host before any HIP call.

The error-path calls pass fake (aligned, never dereferenced) device pointers;
they run only where no GPU is visible, so that a validation bug can never
launch a kernel on them.
"""

import ctypes as C

import numpy as np
import pytest

from paper_2506_01986_amd import specmemo as sm
from paper_2506_01986_amd import synth


def _no_gpu():
    import torch
    return not torch.cuda.is_available()


cpu_only = pytest.mark.skipif(not _no_gpu(), reason="fake device pointers: host validation tests run without a GPU")

FAKE = 1 << 20          # 16-byte aligned, never dereferenced


def test_library_loads_and_exports_every_declared_function():
    lib = sm.load()
    names = sm.declared_functions()
    assert {"specmemo_medusa_topk", "specmemo_tree_attn", "specmemo_accept", "specmemo_kv_compact"} <= set(names)
    for n in names:
        assert hasattr(lib, n), n
    assert sm.abi_version() == 9


class FakeTrees(sm.Trees):
    def __init__(self, trees):
        node_off = np.concatenate([[0], np.cumsum([t.n for t in trees])])
        super().__init__(node_off, np.concatenate([t.parent for t in trees]),
                         np.concatenate([t.depth for t in trees]), np.concatenate([t.rank for t in trees]),
                         dev_arrays=[FAKE, FAKE, FAKE, FAKE])


class FakeKV(sm.KVPool):
    def __init__(self, lens, caps, bases, n_kv=2, d=128, cap_total=None):
        self.k = self.v = self.seq_len = FAKE
        self.seq_base_h = np.asarray(bases, np.int64)
        self.seq_cap_h = np.asarray(caps, np.int32)
        self.seq_len_h = np.asarray(lens, np.int32)
        self.n_kv, self.head_dim = n_kv, d
        self.cap_total = cap_total if cap_total is not None else int(max(np.add(bases, caps)))


def expect(code, fn, *a, **k):
    with pytest.raises(sm.SpecmemoError) as e:
        fn(*a, **k)
    assert e.value.name == code, str(e.value)
    return str(e.value)


def attn(trees, kv, n_q=4, dt=sm.BF16):
    sm.tree_attn(dt, trees, kv, n_q, FAKE, FAKE, ws=FAKE, ws_bytes=1 << 30, stream=0)


def topk(trees, hidden=256, vocab=1000, n_heads=3, k=(4, 2, 2), dt=sm.BF16, ws_bytes=1 << 30, logits=None,
         layout=sm.HEADS_ROWMAJOR):
    sm.medusa_topk(dt, trees, hidden, vocab, n_heads, k, FAKE, FAKE, FAKE, FAKE, FAKE, logits_out=logits,
                   ws=FAKE, ws_bytes=ws_bytes, stream=0, head_layout=layout)


@cpu_only
def test_tree_errors():
    t = synth.t16()
    bad = synth.Tree(t.parent.copy(), t.depth.copy(), t.rank.copy())
    bad.parent[5] = 7                      # parent after child
    msg = expect("E_TREE", topk, FakeTrees([bad]))
    assert "parent" in msg
    dup = synth.Tree(t.parent.copy(), t.depth.copy(), t.rank.copy())
    dup.rank[2] = 0                        # duplicate sibling rank under the root
    expect("E_TREE", topk, FakeTrees([dup]))
    expect("E_TREE", topk, FakeTrees([t]), n_heads=2, k=(4, 2))          # depth 3 > 2 heads
    expect("E_TREE", topk, FakeTrees([t]), k=(3, 2, 2))                 # rank 3 >= top-3
    dep = synth.Tree(t.parent.copy(), t.depth.copy(), t.rank.copy())
    dep.depth[6] = 3
    expect("E_TREE", topk, FakeTrees([dep]))
    big = synth.random_tree(np.random.default_rng(0), 129, max_depth=15, max_kids=30)
    expect("E_TREE", attn, FakeTrees([big]), FakeKV([10], [200], [0]))


@cpu_only
def test_argument_errors():
    t = FakeTrees([synth.t16()])
    expect("E_DTYPE", topk, t, dt=7)
    expect("E_ARG", topk, t, hidden=100)             # not a multiple of 8
    expect("E_ARG", topk, t, k=(4, 2, 0))
    expect("E_ARG", topk, t, k=(40, 2, 2))           # > 32
    expect("E_ARG", topk, t, n_heads=16, k=(4,) * 16)
    expect("E_DTYPE", attn, t, FakeKV([10], [40], [0], d=64))      # bf16 needs d = 128
    expect("E_ARG", attn, t, FakeKV([10], [40], [0], n_kv=3), n_q=4)
    with pytest.raises(sm.SpecmemoError) as e:
        sm.accept(sm.BF16, t, 1000, sm.GREEDY, FAKE, FAKE, FAKE, FAKE, 2, FAKE, stream=0)
    assert e.value.name == "E_ARG" and "path_stride" in str(e.value)
    with pytest.raises(sm.SpecmemoError) as e:
        sm.accept(sm.BF16, t, 1000, sm.TYPICAL, FAKE, FAKE, FAKE, FAKE, 4, FAKE, temperature=0.0, ws=FAKE,
                  ws_bytes=1 << 20, stream=0)
    assert e.value.name == "E_ARG"
    with pytest.raises(sm.SpecmemoError) as e:       # misaligned device pointer
        sm.tree_attn(sm.BF16, t, FakeKV([10], [40], [0]), 4, FAKE + 2, FAKE, stream=0)
    assert e.value.name == "E_ARG"


@cpu_only
def test_packed_head_errors_and_sizes():
    t = FakeTrees([synth.t16()])
    expect("E_ARG", topk, t, layout=7)
    expect("E_DTYPE", topk, t, dt=sm.FP32, layout=sm.HEADS_PACKED)
    assert sm.packed_heads_bytes(sm.BF16, 4, 32000, 8192) == 4 * 500 * 256 * 4096
    assert sm.packed_heads_bytes(sm.BF16, 3, 1000, 72) == 3 * 16 * 3 * 4096     # ragged: 16 row groups, 3 k steps
    assert sm.packed_heads_bytes(sm.FP32, 3, 1000, 256) == 0
    assert sm.packed_heads_bytes(sm.BF16, 3, 1000, 100) == 0                    # hidden % 8 != 0
    with pytest.raises(sm.SpecmemoError) as e:
        sm.pack_heads(sm.FP32, 3, 1000, 256, FAKE, FAKE * 2, stream=0)
    assert e.value.name == "E_DTYPE"
    with pytest.raises(sm.SpecmemoError) as e:
        sm.pack_heads(sm.BF16, 3, 1000, 100, FAKE, FAKE * 2, stream=0)
    assert e.value.name == "E_ARG"
    with pytest.raises(sm.SpecmemoError) as e:                                  # dst overlaps src
        sm.pack_heads(sm.BF16, 3, 1000, 256, FAKE, FAKE + 4096, stream=0)
    assert e.value.name == "E_ARG" and "overlap" in str(e.value)


@cpu_only
def test_budget_errors():
    t = FakeTrees([synth.t16(), synth.t16()])
    expect("E_BUDGET", attn, t, FakeKV([10, 10], [25, 26], [0, 30]))            # 10 + 16 > 25
    expect("E_BUDGET", attn, t, FakeKV([10, 10], [26, 26], [0, 20]))            # slabs overlap
    expect("E_BUDGET", attn, t, FakeKV([10, 10], [26, 26], [0, 30], cap_total=50))
    # a slab base near the int64 limit: base + cap would overflow
    expect("E_BUDGET", attn, t, FakeKV([10, 10], [26, 26], [0, 2 ** 63 - 10], cap_total=100))
    with pytest.raises(sm.SpecmemoError) as e:
        sm.kv_compact(sm.BF16, t, FakeKV([10, 10], [25, 26], [0, 30]), FAKE, FAKE, 5, stream=0)
    assert e.value.name == "E_BUDGET"


@cpu_only
def test_workspace_errors_and_sizes():
    t = FakeTrees([synth.t16()])
    need = sm.workspace_bytes(sm.WS_TOPK, sm.BF16, t, None, 3, 1000)
    assert need >= 1 * 3 * 1000 * 4                           # the fp32 logits
    expect("E_WORKSPACE", topk, t, ws_bytes=1 * 3 * 1000 * 4 - 4)
    # typical: two floats and an int per node; greedy: one int per node (256-byte granules)
    assert sm.workspace_bytes(sm.WS_ACCEPT, sm.BF16, t, None, sm.TYPICAL, 0) == 256 >= 16 * (2 * 4 + 4)
    assert sm.workspace_bytes(sm.WS_ACCEPT, sm.BF16, t, None, sm.GREEDY, 0) == 256 >= 16 * 4
    # more than 32 sequences: the fused acceptance and compaction keeps their descriptors too
    many = FakeTrees([synth.t16()] * 40)
    assert sm.workspace_bytes(sm.WS_ACCEPT, sm.BF16, many, None, sm.GREEDY, 0) == \
        -(-(40 * 16 * 4) // 256) * 256 + -(-(40 * 24) // 256) * 256
    with pytest.raises(sm.SpecmemoError) as e:       # greedy keeps one arg-best token per node
        sm.accept(sm.BF16, t, 1000, sm.GREEDY, FAKE, FAKE, FAKE, FAKE, 4, FAKE, ws=FAKE, ws_bytes=60, stream=0)
    assert e.value.name == "E_WORKSPACE"
    # a long sequence alone on the device is split along its KV range: partials need workspace
    big = FakeTrees([synth.t64()])
    kv = FakeKV([100000], [100064], [0], n_kv=1, d=128)
    assert sm.workspace_bytes(sm.WS_ATTN, sm.BF16, big, kv, 1) > 0
    with pytest.raises(sm.SpecmemoError) as e:
        sm.tree_attn(sm.BF16, big, kv, 1, FAKE, FAKE, ws=FAKE, ws_bytes=16, stream=0)
    assert e.value.name == "E_WORKSPACE"
    assert sm.workspace_bytes(sm.WS_ATTN, 9, big, kv, 1) == 0      # invalid arguments report 0


@cpu_only
def test_last_error_cleared_by_success_is_thread_local():
    import threading
    t = FakeTrees([synth.t16()])
    expect("E_DTYPE", topk, t, dt=7)
    msgs = []
    th = threading.Thread(target=lambda: msgs.append(sm.load().specmemo_last_error()))
    th.start()
    th.join()
    assert msgs == [b""]
    assert sm.load().specmemo_last_error() != b""


@cpu_only
def test_planned_tree_sizes_pass_the_budget_check():
    # Trees cut to the planner's sizes fit their slabs exactly: every host
    # check passes and only the launch fails, as no device is visible; one
    # node more breaks the budget.
    lens, caps = [100, 50, 7, 0], [164, 60, 8, 300]
    sizes = [int(x) for x in sm.plan_tree_sizes(lens, caps, 64)]
    assert sizes == [64, 10, 1, 64]
    bases = np.concatenate([[0], np.cumsum(caps)[:-1]])
    t = synth.t64()

    def cut(n):
        return synth.Tree(t.parent[:n].copy(), t.depth[:n].copy(), t.rank[:n].copy())

    kv = FakeKV(lens, caps, bases)
    expect("E_HIP", attn, FakeTrees([cut(n) for n in sizes]), kv)
    expect("E_BUDGET", attn, FakeTrees([cut(n) for n in sizes[:1]] + [cut(sizes[1] + 1)] + [cut(n) for n in sizes[2:]]),
           kv)


@cpu_only
def test_padded_batching_errors():
    one = synth.tree_from_rank_paths([()])
    t = FakeTrees([synth.t64(), one])                     # the deepest tree has 4 levels
    assert sm.key_mask_words(1) == 4 and sm.key_mask_words(64) == 5 and sm.key_mask_words(65) == 6
    assert sm.key_mask_words(0) == 0

    def pad(kv, ws_bytes=256, key_valid=FAKE, pos=FAKE, words=None):
        sm.kv_pad_update(sm.BF16, t, kv, FAKE, FAKE, 5, key_valid, pos, ws=FAKE, ws_bytes=ws_bytes, stream=0,
                         key_valid_words=sm.key_mask_words(kv.cap_total) if words is None else words)

    roomy = FakeKV([10, 10], [80, 40], [0, 100])
    expect("E_HIP", pad, roomy)                           # every host check passes
    # the single-node slab holds its tree (36 + 1 <= 38) but not a uniform
    # length of up to 5 rows (36 + 5 > 38); compaction accepts the same pool
    tight = FakeKV([10, 36], [80, 38], [0, 100])
    expect("E_BUDGET", pad, tight)
    expect("E_HIP", sm.kv_compact, sm.BF16, t, tight, FAKE, FAKE, 5, stream=0)
    expect("E_WORKSPACE", pad, roomy, ws_bytes=2)
    expect("E_ARG", pad, roomy, key_valid=None)
    expect("E_ARG", pad, roomy, pos=None)
    expect("E_ARG", pad, roomy, words=sm.key_mask_words(roomy.cap_total) - 1)   # a flag array too short
    with pytest.raises(sm.SpecmemoError) as e:
        sm.tree_attn_padded(sm.BF16, t, roomy, None, 4, FAKE, FAKE, ws=FAKE, ws_bytes=1 << 30, stream=0,
                            key_valid_words=1 << 20)
    assert e.value.name == "E_ARG"
    with pytest.raises(sm.SpecmemoError) as e:
        sm.tree_attn_padded(sm.BF16, t, roomy, FAKE, 4, FAKE, FAKE, ws=FAKE, ws_bytes=1 << 30, stream=0,
                            key_valid_words=3)
    assert e.value.name == "E_ARG" and "words" in str(e.value)
    assert sm.workspace_bytes(sm.WS_PAD, sm.BF16, t, None, 0) >= 4


@cpu_only
def test_projection_resblock_and_sampling_errors():
    def logits(**k):
        a = dict(dt=sm.BF16, B=2, hidden=64, vocab=100, n_heads=2, h=FAKE, head_w=FAKE, logits_out=FAKE,
                 head_layout=sm.HEADS_PACKED)
        a.update(k)
        sm.head_logits(a["dt"], a["B"], a["hidden"], a["vocab"], a["n_heads"], a["h"], a["head_w"], a["logits_out"],
                       head_layout=a["head_layout"], stream=0)
    expect("E_HIP", logits)                                     # every host check passes
    expect("E_DTYPE", logits, dt=sm.FP32)                       # packed heads are bf16 only
    expect("E_ARG", logits, head_layout=4)
    expect("E_ARG", logits, hidden=60)
    expect("E_ARG", logits, B=0)
    expect("E_ARG", logits, logits_out=None)
    expect("E_HIP", logits, head_layout=sm.HEADS_PACKED | sm.HEADS_INPUT_PER_HEAD)
    expect("E_ARG", sm.medusa_resblock, sm.BF16, 2, 64, 2, FAKE, FAKE, FAKE, FAKE, w1_layout=sm.HEADS_ROWMAJOR, stream=0)
    expect("E_DTYPE", sm.medusa_resblock, sm.FP32, 2, 64, 2, FAKE, FAKE, FAKE, FAKE, w1_layout=sm.HEADS_PACKED,
           stream=0)
    t = FakeTrees([synth.t16()])
    for temp in (0.0, -1.0, float("inf"), 1e-45):
        expect("E_ARG", sm.sample_next, sm.BF16, t, 100, temp, 1, 0, FAKE, FAKE, FAKE, 4, FAKE, stream=0)
    expect("E_ARG", sm.sample_next, sm.BF16, t, 100, 1.0, 1, 0, FAKE, FAKE, FAKE, 3, FAKE, stream=0)   # stride < depth + 1
    expect("E_HIP", sm.sample_next, sm.BF16, t, 100, 1.0, 1, 0, FAKE, FAKE, FAKE, 4, FAKE, stream=0)
    # the segmented form: one 64-bit word per 1024-token segment of each row
    need = sm.workspace_bytes(sm.WS_SAMPLE, sm.BF16, t, None, 0, 32000)
    assert need >= 1 * 32 * 8 and need % 256 == 0
    assert sm.workspace_bytes(sm.WS_SAMPLE, sm.BF16, t, None, 0, 0) == 0
    expect("E_WORKSPACE", sm.sample_next, sm.BF16, t, 32000, 1.0, 1, 0, FAKE, FAKE, FAKE, 4, FAKE, ws=FAKE,
           ws_bytes=need - 8, stream=0)
    expect("E_HIP", sm.sample_next, sm.BF16, t, 32000, 1.0, 1, 0, FAKE, FAKE, FAKE, 4, FAKE, ws=FAKE, ws_bytes=need,
           stream=0)


@cpu_only
def test_fused_acceptance_and_compaction_errors():
    # the fused call takes the checks of both calls: acceptance first, then the pool
    t = FakeTrees([synth.t16(), synth.t16()])

    def fused(kv, mode=sm.GREEDY, stride=4, ws_bytes=1 << 20, **kw):
        sm.accept_compact(sm.BF16, t, kv, 1000, mode, FAKE, FAKE, FAKE, FAKE, stride, FAKE, ws=FAKE,
                          ws_bytes=ws_bytes, stream=0, **kw)
    ok_kv = FakeKV([10, 10], [26, 26], [0, 30])
    assert "path_stride" in expect("E_ARG", fused, ok_kv, stride=2)
    expect("E_WORKSPACE", fused, ok_kv, ws_bytes=4 * 31)                  # one int32 per node: 32 needed
    expect("E_WORKSPACE", fused, ok_kv, mode=sm.TYPICAL, ws_bytes=4 * 32)  # typical: two floats and an int per node
    expect("E_ARG", fused, ok_kv, mode=sm.TYPICAL, temperature=-1.0)
    expect("E_BUDGET", fused, FakeKV([10, 10], [25, 26], [0, 30]))       # 10 + 16 > 25
    expect("E_BUDGET", fused, FakeKV([10, 10], [26, 26], [0, 20]))       # slabs overlap
    bad = FakeKV([10, 10], [26, 26], [0, 30])
    bad.seq_len = FAKE + 2                                                # misaligned device seq_len
    expect("E_ARG", fused, bad)
    expect("E_DTYPE", fused, FakeKV([10, 10], [26, 26], [0, 30], d=64))   # bf16 needs d = 128


@cpu_only
def test_noalloc_attention_checks_and_scratch_limit():
    """The allocation-free attention call validates like the workspace form,
    and a split that would need more than the static scratch is rejected
    before any HIP call (a fixed 64-key chunk over long sequences: the
    tuning variable is read once per process, so the check runs in a child)."""
    import os
    import subprocess
    import sys
    bad = synth.Tree(synth.t16().parent.copy(), synth.t16().depth.copy(), synth.t16().rank.copy())
    bad.parent[5] = 7
    expect("E_TREE", sm.tree_attn_noalloc, sm.BF16, FakeTrees([bad]), FakeKV([10], [100], [0], d=128), 4, FAKE, FAKE)
    expect("E_ARG", sm.tree_attn_noalloc, sm.BF16, FakeTrees([synth.t16()]), FakeKV([10], [100], [0]), 3, FAKE, FAKE)
    expect("E_BUDGET", sm.tree_attn_noalloc, sm.BF16, FakeTrees([synth.t16()]), FakeKV([90], [100], [0]), 4, FAKE,
           FAKE)
    child = (
        "import numpy as np\n"
        "from tests import test_abi_cpu as t\n"
        "from paper_2506_01986_amd import specmemo as sm, synth\n"
        "trees = t.FakeTrees([synth.t64()] * 4)\n"
        "kv = t.FakeKV([1 << 22] * 4, [(1 << 22) + 64] * 4, [i * ((1 << 22) + 64) for i in range(4)], n_kv=8)\n"
        "need = sm.workspace_bytes(sm.WS_ATTN, sm.BF16, trees, kv, 64)\n"
        "assert need > sm.STATIC_SCRATCH_BYTES, need\n"
        "msg = t.expect('E_WORKSPACE', sm.tree_attn_noalloc, sm.BF16, trees, kv, 64, t.FAKE, t.FAKE)\n"
        "assert 'static scratch' in msg, msg\n"
        "print('ok', need)\n")
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, "-c", child], cwd=root, capture_output=True, text=True, timeout=120,
                       env={**os.environ, "SPECMEMO_ATTN_CHUNK": "64", "HIP_VISIBLE_DEVICES": ""})
    assert r.returncode == 0 and r.stdout.startswith("ok"), r.stdout + r.stderr
