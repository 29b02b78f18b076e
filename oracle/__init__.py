"""CPU oracle of the tree-verification step.  TEST INFRASTRUCTURE.

A ctypes binding over ``specmemo_oracle.c`` (fp64 loops, OpenMP).  Only the
tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py``
may import this package.  It never imports the HIP library or its binding.

Every function takes stored arrays (float32, or uint16 bf16 bit patterns) and
widens them exactly to float64.  Which passage of SpecMemo each stage follows
is stated in the C source.
"""

from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "specmemo_oracle.c")
LIB = os.path.join(HERE, "_build", "liboracle.so")

_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (-O2, no fast-math, OpenMP)."""
    if force or not os.path.exists(LIB):
        os.makedirs(os.path.dirname(LIB), exist_ok=True)
        tmp = LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared",
                               "-o", tmp, SRC, "-lm"])
        os.replace(tmp, LIB)
    return LIB


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build()
        _lib = C.CDLL(LIB)
    return _lib


def threads(n: int = 0) -> int:
    """Threads of the oracle's parallel loops: n >= 1 sets them; returns the
    count in use."""
    return int(lib().oracle_threads(int(n)))


def _dt(x: np.ndarray) -> int:
    if x.dtype == np.float32:
        return 0
    if x.dtype == np.uint16:
        return 1
    raise TypeError(f"stored arrays are float32 or uint16 (bf16 bits), got {x.dtype}")


def _p(x: np.ndarray):
    assert x.flags["C_CONTIGUOUS"], "oracle inputs must be C-contiguous"
    return x.ctypes.data_as(C.c_void_p)


def _i32(x) -> np.ndarray:
    return np.ascontiguousarray(x, dtype=np.int32)


def head_logits(h: np.ndarray, W: np.ndarray, bsel=None) -> np.ndarray:
    """z[s, i, v] = sum_c W[i, v, c] * h[b_s, c] in float64 (``bsel``: batch rows)."""
    B, hidden = h.shape
    n_heads, vocab, hid2 = W.shape
    assert hid2 == hidden and _dt(h) == _dt(W)
    bs = None if bsel is None else _i32(bsel)
    nb = B if bs is None else len(bs)
    z = np.empty((nb, n_heads, vocab), dtype=np.float64)
    lib().oracle_head_logits(_dt(h), B, hidden, vocab, n_heads, _p(h), _p(W),
                             0 if bs is None else len(bs), None if bs is None else _p(bs), _p(z))
    return z


def topk(z: np.ndarray, k: int):
    """Top-k of each row of a float64 [rows, vocab] array: (ids, values),
    larger value first, ties to the lower id."""
    z = np.ascontiguousarray(z, dtype=np.float64)
    rows, vocab = z.reshape(-1, z.shape[-1]).shape
    ids = np.empty((rows, k), dtype=np.int32)
    vals = np.empty((rows, k), dtype=np.float64)
    lib().oracle_topk(rows, vocab, k, _p(z), _p(ids), _p(vals))
    return ids.reshape(z.shape[:-1] + (k,)), vals.reshape(z.shape[:-1] + (k,))


def heads_topk(z: np.ndarray, topk_per_head, kmax: int):
    """Per-head top-k of z[B, n_heads, vocab] into [B, n_heads, kmax] (-1 padded)."""
    B, n_heads, _ = z.shape
    ids = np.full((B, n_heads, kmax), -1, dtype=np.int32)
    vals = np.full((B, n_heads, kmax), -np.inf, dtype=np.float64)
    for i in range(n_heads):
        k = int(topk_per_head[i])
        a, v = topk(z[:, i, :], k)
        ids[:, i, :k] = a
        vals[:, i, :k] = v
    return ids, vals


def tree_tokens(node_off, depth, rank, root_tok, topk_ids) -> np.ndarray:
    B, n_heads, kmax = topk_ids.shape
    node_off, depth, rank, root_tok = map(_i32, (node_off, depth, rank, root_tok))
    ids = _i32(topk_ids)
    out = np.empty(int(node_off[-1]), dtype=np.int32)
    lib().oracle_tree_tokens(B, _p(node_off), _p(depth), _p(rank), _p(root_tok), n_heads, kmax,
                             _p(ids), _p(out))
    return out


def tree_attn(q, K, V, node_off, parent, seq_len, seq_base, n_kv: int, scale: float | None = None,
              sel=None, key_valid=None) -> np.ndarray:
    """Tree-masked attention in float64.

    q: [sumN, n_q, d]; K, V: pool [n_kv, cap_total, d]; sel: optional array of
    (global node, q head) pairs; key_valid: optional [cap_total] flags, 0 for
    a cached pad token (padded batching).  Returns [sumN, n_q, d] or
    [len(sel), d].
    """
    sumN, n_q, d = q.shape
    assert K.shape == V.shape and K.shape[0] == n_kv and K.shape[2] == d
    assert _dt(q) == _dt(K) == _dt(V)
    node_off, parent, seq_len = map(_i32, (node_off, parent, seq_len))
    seq_base = np.ascontiguousarray(seq_base, dtype=np.int64)
    scale = 1.0 / np.sqrt(d) if scale is None else float(scale)
    B = len(node_off) - 1
    kvf = None
    if key_valid is not None:
        kvf = np.ascontiguousarray(np.asarray(key_valid) != 0, dtype=np.uint8)
        assert kvf.shape == (K.shape[1],)
    kvp = _p(kvf) if kvf is not None else None
    if sel is None:
        out = np.empty((sumN, n_q, d), dtype=np.float64)
        lib().oracle_tree_attn(_dt(q), B, _p(node_off), _p(parent), _p(seq_len), _p(seq_base),
                               n_q, n_kv, d, C.c_int64(K.shape[1]), C.c_double(scale), _p(q),
                               _p(K), _p(V), 0, None, _p(out), kvp)
    else:
        s = _i32(sel).reshape(-1, 2)
        out = np.empty((len(s), d), dtype=np.float64)
        lib().oracle_tree_attn(_dt(q), B, _p(node_off), _p(parent), _p(seq_len), _p(seq_base),
                               n_q, n_kv, d, C.c_int64(K.shape[1]), C.c_double(scale), _p(q),
                               _p(K), _p(V), len(s), _p(s), _p(out), kvp)
    return out


def accept_greedy(logits, node_tok, node_off, parent, depth, path_stride: int):
    sumN, vocab = logits.shape
    node_off, parent, depth, node_tok = map(_i32, (node_off, parent, depth, node_tok))
    B = len(node_off) - 1
    acc = np.empty(B, np.int32)
    path = np.empty((B, path_stride), np.int32)
    nxt = np.empty(B, np.int32)
    lib().oracle_accept_greedy(_dt(logits), B, _p(node_off), _p(parent), _p(depth), vocab,
                               _p(logits), _p(node_tok), path_stride, _p(acc), _p(path), _p(nxt))
    return acc, path, nxt


def accept_typical(logits, node_tok, node_off, parent, depth, path_stride: int,
                   temperature: float, eps: float, delta: float, edges: bool = False):
    sumN, vocab = logits.shape
    node_off, parent, depth, node_tok = map(_i32, (node_off, parent, depth, node_tok))
    B = len(node_off) - 1
    acc = np.empty(B, np.int32)
    path = np.empty((B, path_stride), np.int32)
    nxt = np.empty(B, np.int32)
    lp = np.full(sumN, np.nan)
    lt = np.full(sumN, np.nan)
    lib().oracle_accept_typical(_dt(logits), B, _p(node_off), _p(parent), _p(depth), vocab,
                                _p(logits), _p(node_tok), C.c_double(temperature), C.c_double(eps),
                                C.c_double(delta), path_stride, _p(acc), _p(path), _p(nxt),
                                _p(lp), _p(lt))
    if edges:
        return acc, path, nxt, lp, lt
    return acc, path, nxt


def softmax_stats(logits, temperature: float):
    """(lse, H) of each row x = z / T in float64: log sum exp x and the
    entropy of softmax(x)."""
    rows, vocab = logits.shape
    lse = np.empty(rows, np.float64)
    ent = np.empty(rows, np.float64)
    lib().oracle_softmax_stats(_dt(logits), rows, vocab, _p(np.ascontiguousarray(logits)),
                               C.c_double(temperature), _p(lse), _p(ent))
    return lse, ent


def kv_compact(K, V, seq_base, seq_len, accept_len, path):
    """In-place compaction on host copies of the pool; returns the new seq_len."""
    n_kv, cap_total, d = K.shape
    assert K.dtype == V.dtype and K.flags["C_CONTIGUOUS"] and V.flags["C_CONTIGUOUS"]
    seq_base = np.ascontiguousarray(seq_base, dtype=np.int64)
    sl = _i32(seq_len).copy()
    acc, path = _i32(accept_len), _i32(path)
    B, stride = path.shape
    lib().oracle_kv_compact(K.dtype.itemsize, B, n_kv, d, C.c_int64(cap_total), _p(K), _p(V),
                            _p(seq_base), _p(sl), _p(acc), _p(path), stride)
    return sl


def resblock(h, W1, b1) -> np.ndarray:
    """Medusa residual blocks in float64: [n_heads, B, hidden] of
    h + SiLU(W1_i h + b1_i) (the blocks' outputs before storage rounding)."""
    B, hidden = h.shape
    n_heads = W1.shape[0]
    assert W1.shape == (n_heads, hidden, hidden) and b1.shape == (n_heads, hidden)
    assert _dt(h) == _dt(W1) == _dt(b1)
    out = np.empty((n_heads, B, hidden), dtype=np.float64)
    lib().oracle_resblock(_dt(h), B, hidden, n_heads, _p(h), _p(W1), _p(b1), _p(out))
    return out


def to_storage(x: np.ndarray, dtype: str) -> np.ndarray:
    """float64 -> the storage type, as a kernel stores an fp32 result: rounded
    to float32 (nearest even), then for bf16 to its top 16 bits (nearest even)."""
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    if dtype == "fp32":
        return f
    u = f.view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    return r


def philox4x64_10(ctr, key) -> np.ndarray:
    """Philox4x64-10 blocks: ctr [n, 4], key [n, 2] (uint64) -> [n, 4]."""
    c = np.ascontiguousarray(ctr, dtype=np.uint64).reshape(-1, 4)
    k = np.ascontiguousarray(key, dtype=np.uint64).reshape(-1, 2)
    assert len(c) == len(k)
    out = np.empty_like(c)
    lib().oracle_philox4x64_10(len(c), _p(c), _p(k), _p(out))
    return out


def gumbel(words) -> np.ndarray:
    """Standard Gumbel values -log(-log u) of 64-bit random words, with
    u = (top 23 bits + 1/2) / 2^23, in float64."""
    x = np.ascontiguousarray(words, dtype=np.uint64).reshape(-1)
    g = np.empty(len(x), np.float64)
    lib().oracle_gumbel(len(x), _p(x), _p(g))
    return g


def sample_next(logits, node_off, accept_len, path, temperature: float, seed: int, offset: int):
    """Gumbel-max draw from softmax(z / T) of each sequence's last accepted
    node, keys in float64.  Returns (next_tok, best key, second-best key) of
    each sequence."""
    sumN, vocab = logits.shape
    node_off, acc, path = _i32(node_off), _i32(accept_len), _i32(path)
    B, stride = path.shape
    tok = np.empty(B, np.int32)
    best, second = np.empty(B, np.float64), np.empty(B, np.float64)
    inv_t = np.float32(1.0) / np.float32(temperature)
    lib().oracle_sample_next(_dt(logits), B, _p(node_off), vocab, C.c_float(inv_t), C.c_uint64(seed),
                             C.c_uint64(offset), _p(logits), _p(acc), _p(path), stride, _p(tok), _p(best),
                             _p(second))
    return tok, best, second
