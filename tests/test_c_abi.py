"""The C ABI from C: the header compiles as strict C99 and as C++, and a plain
C program (tests/c/verify_step.c) that allocates device memory with the HIP
runtime's C API runs one verify step through the library (the four stage
calls, or three with acceptance and compaction fused); its outputs match the
oracle's to the same bar as the Python-driven parity tests."""

import os
import subprocess

import numpy as np
import pytest

import oracle
from tests import ties
from paper_2506_01986_amd import configs, specmemo as sm, synth

HERE = os.path.dirname(os.path.abspath(__file__))
INCLUDE = os.path.join(os.path.dirname(HERE), "include")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
TOL = {"fp32": (1e-5, 1e-5), "bf16": (1e-2, 2e-2)}


def _compile(args, cwd):
    r = subprocess.run(args, cwd=cwd, capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr[-4000:]


@pytest.mark.parametrize("lang", ["c99", "c++17"])
def test_header_is_strict_c99_and_cxx(tmp_path, lang):
    src = tmp_path / "h.c"
    src.write_text('#include "specmemo.h"\n'
                   "int main(void) { return specmemo_abi_version() == SPECMEMO_ABI_VERSION ? 0 : 1; }\n")
    cc = ["gcc", "-std=c99"] if lang == "c99" else ["g++", "-std=c++17", "-x", "c++"]
    _compile(cc + ["-Wall", "-Wextra", "-Werror", "-pedantic", "-I", INCLUDE, "-c", str(src), "-o", "h.o"], tmp_path)


def build_consumer(out_dir) -> str:
    exe = os.path.join(str(out_dir), "verify_step")
    libdir = os.path.dirname(sm.LIB_PATH)
    _compile(["gcc", "-std=c99", "-O2", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
              "-I", os.path.join(ROCM, "include"), "-I", INCLUDE, os.path.join(HERE, "c", "verify_step.c"),
              "-o", exe, "-L", libdir, "-lspecmemo", "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
              f"-Wl,-rpath,{libdir}", f"-Wl,-rpath,{os.path.join(ROCM, 'lib')}"], out_dir)
    return exe


def test_c_consumer_builds_and_links(tmp_path):
    sm.load()
    assert os.path.exists(build_consumer(tmp_path))


def _workload(dtype):
    cfg = configs.Config(name="c_abi", dtype=dtype, B=3, n_q=8, n_kv=2, head_dim=64 if dtype == "fp32" else 128,
                         hidden=96, vocab=700, n_heads=3, topk=(6, 4, 3), tree="T16", kv_len=(1, 1), seed=31,
                         w_std=1.0 if dtype == "fp32" else 0.05, p_accept=0.8)
    rng = np.random.default_rng(31)
    # a random tree, a single root, and a root with six children (the widest level)
    trees = [synth.random_tree(rng, 30, max_depth=3, max_kids=3), synth.tree_from_rank_paths([()]),
             synth.tree_from_rank_paths([()] + [(r,) for r in range(6)])]
    return synth.make(cfg, trees=trees, lens=[70, 0, 300])


@pytest.mark.gpu
@pytest.mark.parametrize("fused", [False, True], ids=["four_calls", "accept_compact"])
@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_c_program_verify_step_matches_the_oracle(tmp_path, dtype, fused):
    sm.load()
    exe = build_consumer(tmp_path)
    wl = _workload(dtype)
    cfg = wl.cfg
    stride = cfg.n_heads + 1
    z64, _ = ties.guard_hidden(wl)          # no near-tied top-k logits: ids compare exactly
    ids64, _ = oracle.heads_topk(z64, cfg.topk, cfg.kmax)
    tok64 = oracle.tree_tokens(wl.node_off, wl.depth, wl.rank, wl.root_tok, ids64)
    lg = synth.planted_logits(wl, tok64)
    d = tmp_path
    (d / "meta.txt").write_text(" ".join(str(x) for x in (
        0 if dtype == "fp32" else 1, cfg.B, cfg.hidden, cfg.vocab, cfg.n_heads, cfg.n_q, cfg.n_kv, cfg.head_dim,
        wl.cap_total, stride, *cfg.topk)) + "\n")
    for name, arr in (("node_off", wl.node_off), ("parent", wl.parent), ("depth", wl.depth), ("rank", wl.rank),
                      ("seq_base", wl.seq_base.astype(np.int64)), ("seq_len", wl.lens), ("seq_cap", wl.seq_cap),
                      ("k", wl.pool_k), ("v", wl.pool_v), ("h", wl.hidden), ("head_w", wl.head_w), ("q", wl.q),
                      ("base_logits", lg), ("root_tok", wl.root_tok)):
        (d / f"{name}.bin").write_bytes(np.ascontiguousarray(arr).tobytes())
    print(f"[c_abi] {dtype} fused={fused}: B={cfg.B} sumN={wl.total_nodes} L={wl.lens.tolist()}", flush=True)
    r = subprocess.run([exe, str(d)] + (["fused"] if fused else []), capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    store = np.float32 if dtype == "fp32" else np.uint16

    def out(name, dt, shape):
        return np.fromfile(d / f"out_{name}.bin", dtype=dt).reshape(shape)

    B, N = cfg.B, wl.total_nodes
    atol, rtol = TOL[dtype]
    # (a) logits within tolerance, top-k ids and tree tokens exact
    z = out("logits", np.float32, (B, cfg.n_heads, cfg.vocab))
    assert np.all(np.abs(z - z64) <= atol + rtol * np.abs(z64))
    assert np.array_equal(out("topk_ids", np.int32, (B, cfg.n_heads, cfg.kmax)), ids64)
    assert np.array_equal(out("node_tok", np.int32, (N,)), tok64)
    # (b) attention: every (node, head) row
    att = synth.storage_to_f64(out("attn", store, (N, cfg.n_q, cfg.head_dim)), dtype)
    ref = oracle.tree_attn(wl.q, wl.pool_k, wl.pool_v, wl.node_off, wl.parent, wl.lens, wl.seq_base, cfg.n_kv)
    assert np.all(np.abs(att - ref) <= atol + rtol * np.abs(ref))
    # (c) greedy acceptance of the planted walks, bit-exact
    ra, rp, rn = oracle.accept_greedy(lg, tok64, wl.node_off, wl.parent, wl.depth, stride)
    acc = out("accept_len", np.int32, (B,))
    path = out("path", np.int32, (B, stride))
    assert np.array_equal(acc, ra) and np.array_equal(path, rp)
    assert np.array_equal(out("next_tok", np.int32, (B,)), rn)
    for b in range(B):
        assert path[b, :acc[b] + 1].tolist() == wl.plan_path[b]
    # (d) compaction, bit-exact over the whole pool
    K0, V0 = wl.pool_k.copy(), wl.pool_v.copy()
    new_len = oracle.kv_compact(K0, V0, wl.seq_base, wl.lens, ra, rp)
    assert np.array_equal(out("k", store, K0.shape).view(np.uint8), K0.view(np.uint8))
    assert np.array_equal(out("v", store, V0.shape).view(np.uint8), V0.view(np.uint8))
    assert np.array_equal(out("seq_len", np.int32, (B,)), new_len)
