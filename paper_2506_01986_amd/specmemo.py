"""ctypes binding of libspecmemo (include/specmemo.h).

Argument marshalling only: torch tensors provide device memory and the stream,
numpy arrays the host mirrors; every stage runs in the library's HIP kernels.
The library is loaded on first use; if it has not been built, ``load()``
raises instead of falling back to anything else.
"""

from __future__ import annotations

import ctypes as C
import os
import re
from typing import Optional, Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "_build", "libspecmemo.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "specmemo.h")

FP32, BF16 = 0, 1
GREEDY, TYPICAL = 0, 1
HEADS_ROWMAJOR, HEADS_PACKED, HEADS_INPUT_PER_HEAD = 0, 1, 2
WS_TOPK, WS_ATTN, WS_ACCEPT, WS_PAD, WS_SAMPLE = 0, 1, 2, 3, 4

STATUS = {0: "OK", -1: "E_ARG", -2: "E_DTYPE", -3: "E_TREE", -4: "E_BUDGET", -5: "E_WORKSPACE", -6: "E_HIP"}


class SpecmemoError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{STATUS.get(code, code)}: {msg}")
        self.code = code
        self.name = STATUS.get(code, str(code))


class _Trees(C.Structure):
    _fields_ = [("B", C.c_int32), ("node_off", C.c_void_p), ("parent", C.c_void_p), ("depth", C.c_void_p),
                ("rank", C.c_void_p), ("node_off_h", C.c_void_p), ("parent_h", C.c_void_p),
                ("depth_h", C.c_void_p), ("rank_h", C.c_void_p)]


class _KV(C.Structure):
    _fields_ = [("k", C.c_void_p), ("v", C.c_void_p), ("cap_total", C.c_int64), ("n_kv", C.c_int32),
                ("head_dim", C.c_int32), ("seq_len", C.c_void_p), ("seq_base_h", C.c_void_p),
                ("seq_cap_h", C.c_void_p), ("seq_len_h", C.c_void_p)]


class _Budget(C.Structure):
    _fields_ = [("max_memory", C.c_int64), ("base_model_bytes", C.c_int64), ("head_bytes", C.c_int64),
                ("layers", C.c_int32), ("n_kv", C.c_int32), ("head_dim", C.c_int32), ("vocab", C.c_int32),
                ("elem_bytes", C.c_int32), ("batch", C.c_int32), ("query_count", C.c_int32),
                ("query_length", C.c_int32), ("default_heads", C.c_int32)]


class _BudgetPlan(C.Structure):
    _fields_ = [("kind", C.c_int32), ("heads", C.c_int32), ("nodes", C.c_int32), ("leaves", C.c_int32),
                ("kv_bytes", C.c_int64), ("total_bytes", C.c_int64)]


PLAN_DEFAULT, PLAN_PRUNED, PLAN_FEWER_HEADS, PLAN_NONE = 0, 1, 2, -1

_lib = None


def load():
    """Load libspecmemo.so; raise if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"libspecmemo is not built ({LIB_PATH}); run __graft_entry__.build()")
        lib = C.CDLL(LIB_PATH)
        vp, i32, sz, f32 = C.c_void_p, C.c_int32, C.c_size_t, C.c_float
        PT, PK = C.POINTER(_Trees), C.POINTER(_KV)
        lib.specmemo_medusa_topk.argtypes = [i32, PT, i32, i32, i32, vp, vp, vp, i32, vp, vp, vp, vp, vp, vp, sz, vp]
        lib.specmemo_pack_heads.argtypes = [i32, i32, i32, i32, vp, vp, vp]
        lib.specmemo_pack_heads.restype = C.c_int
        lib.specmemo_packed_heads_bytes.argtypes = [i32, i32, i32, i32]
        lib.specmemo_packed_heads_bytes.restype = C.c_size_t
        lib.specmemo_tree_attn.argtypes = [i32, PT, PK, i32, f32, vp, vp, vp, sz, vp]
        lib.specmemo_tree_attn_noalloc.argtypes = [i32, PT, PK, i32, f32, vp, vp, vp]
        lib.specmemo_accept.argtypes = [i32, PT, i32, i32, f32, f32, f32, vp, vp, vp, vp, i32, vp, vp, sz, vp]
        lib.specmemo_kv_compact.argtypes = [i32, PT, PK, vp, vp, i32, vp]
        lib.specmemo_accept_compact.argtypes = [i32, PT, PK, i32, i32, f32, f32, f32, vp, vp, vp, vp, i32, vp, vp, sz, vp]
        lib.specmemo_workspace_bytes.argtypes = [i32, i32, PT, PK, i32, i32]
        lib.specmemo_workspace_bytes.restype = C.c_size_t
        lib.specmemo_last_error.restype = C.c_char_p
        lib.specmemo_abi_version.restype = C.c_int32
        for f in ("specmemo_medusa_topk", "specmemo_tree_attn", "specmemo_accept", "specmemo_kv_compact",
                  "specmemo_accept_compact", "specmemo_tree_attn_noalloc"):
            getattr(lib, f).restype = C.c_int
        i64 = C.c_int64
        u64 = C.c_uint64
        lib.specmemo_head_logits.argtypes = [i32, i32, i32, i32, i32, vp, vp, i32, vp, vp]
        lib.specmemo_head_logits.restype = C.c_int
        lib.specmemo_medusa_resblock.argtypes = [i32, i32, i32, i32, vp, vp, i32, vp, vp, vp]
        lib.specmemo_medusa_resblock.restype = C.c_int
        lib.specmemo_sample_next.argtypes = [i32, PT, i32, f32, u64, u64, vp, vp, vp, i32, vp, vp, sz, vp]
        lib.specmemo_sample_next.restype = C.c_int
        lib.specmemo_key_mask_words.argtypes = [i64]
        lib.specmemo_key_mask_words.restype = i64
        lib.specmemo_tree_attn_padded.argtypes = [i32, PT, PK, vp, i64, i32, f32, vp, vp, vp, sz, vp]
        lib.specmemo_tree_attn_padded.restype = C.c_int
        lib.specmemo_kv_pad_update.argtypes = [i32, PT, PK, vp, vp, i32, vp, i64, vp, vp, sz, vp]
        lib.specmemo_kv_pad_update.restype = C.c_int
        lib.specmemo_mem_kv_bytes.argtypes = [i32, i32, i32, i32, i64, i32]
        lib.specmemo_mem_buffer_bytes.argtypes = [i32, i32, i32, i32, i32, i32]
        lib.specmemo_mem_total_bytes.argtypes = [i64, i64, i32, i64, i64]
        lib.specmemo_tree_full_nodes.argtypes = [i32, i32]
        for f in ("specmemo_mem_kv_bytes", "specmemo_mem_buffer_bytes", "specmemo_mem_total_bytes",
                  "specmemo_tree_full_nodes"):
            getattr(lib, f).restype = i64
        lib.specmemo_tree_build.argtypes = [i32, i32, i32, i32, vp, vp, vp]
        lib.specmemo_tree_build.restype = C.c_int
        lib.specmemo_tree_leaves.argtypes = [i32, vp, vp, vp]
        lib.specmemo_tree_leaves.restype = i32
        lib.specmemo_tree_prune.argtypes = [i32, vp, vp, vp, i32, vp, vp, vp, vp, vp]
        lib.specmemo_tree_prune.restype = C.c_int
        lib.specmemo_plan_budget.argtypes = [C.POINTER(_Budget), i32, vp, vp, vp, C.POINTER(_BudgetPlan)]
        lib.specmemo_plan_budget.restype = C.c_int
        lib.specmemo_plan_tree_sizes.argtypes = [i32, vp, vp, i32, vp]
        lib.specmemo_plan_tree_sizes.restype = C.c_int
        _lib = lib
    return _lib


def declared_functions() -> list:
    """Names of the functions include/specmemo.h declares."""
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(specmemo_\w+)\s*\(", text)))


def _check(rc: int):
    if rc != 0:
        raise SpecmemoError(rc, load().specmemo_last_error().decode())


def _ptr(x) -> Optional[int]:
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if isinstance(x, np.ndarray):
        return x.ctypes.data
    return x.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        if not torch.cuda.is_available():
            return None
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _i32(x) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(x, dtype=np.int32))


class Trees:
    """Ragged batch of candidate trees: device arrays plus host mirrors."""

    def __init__(self, node_off, parent, depth, rank, device=None, dev_arrays=None):
        self.node_off_h, self.parent_h = _i32(node_off), _i32(parent)
        self.depth_h, self.rank_h = _i32(depth), _i32(rank)
        self.B = len(self.node_off_h) - 1
        if dev_arrays is not None:
            self.dev = dev_arrays
        else:
            import torch
            self.dev = [torch.from_numpy(a.copy()).to(device) for a in
                        (self.node_off_h, self.parent_h, self.depth_h, self.rank_h)]

    @property
    def total_nodes(self) -> int:
        return int(self.node_off_h[-1])

    @property
    def max_depth(self) -> int:
        return int(self.depth_h.max())

    def struct(self) -> _Trees:
        return _Trees(self.B, *[_ptr(t) for t in self.dev],
                      *[a.ctypes.data for a in (self.node_off_h, self.parent_h, self.depth_h, self.rank_h)])


class KVPool:
    """One layer's budget-capped KV pool: device K, V and seq_len, host mirrors."""

    def __init__(self, k, v, seq_len_dev, seq_base, seq_cap, seq_len):
        self.k, self.v, self.seq_len = k, v, seq_len_dev
        self.seq_base_h = np.ascontiguousarray(seq_base, dtype=np.int64)
        self.seq_cap_h = _i32(seq_cap)
        self.seq_len_h = _i32(seq_len)
        self.n_kv, self.cap_total, self.head_dim = (int(s) for s in k.shape)

    def struct(self) -> _KV:
        return _KV(_ptr(self.k), _ptr(self.v), self.cap_total, self.n_kv, self.head_dim,
                   _ptr(self.seq_len), self.seq_base_h.ctypes.data, self.seq_cap_h.ctypes.data,
                   self.seq_len_h.ctypes.data)


def abi_version() -> int:
    return load().specmemo_abi_version()


def workspace_bytes(which: int, dt: int, trees: Trees, kv: Optional[KVPool], n_q_or_heads: int, vocab: int = 0) -> int:
    ts = trees.struct()
    ks = kv.struct() if kv is not None else None
    return load().specmemo_workspace_bytes(which, dt, C.byref(ts), C.byref(ks) if ks is not None else None,
                                           n_q_or_heads, vocab)


def medusa_topk(dt: int, trees: Trees, hidden: int, vocab: int, n_heads: int, topk: Sequence[int], h, head_w,
                root_tok, topk_ids, node_tok, logits_out=None, topk_vals=None, ws=None, ws_bytes: int = 0,
                stream=None, head_layout: int = HEADS_ROWMAJOR):
    ts = trees.struct()
    tk = _i32(topk)
    _check(load().specmemo_medusa_topk(dt, C.byref(ts), hidden, vocab, n_heads, tk.ctypes.data, _ptr(h),
                                       _ptr(head_w), head_layout, _ptr(root_tok), _ptr(logits_out),
                                       _ptr(topk_ids), _ptr(topk_vals), _ptr(node_tok), _ptr(ws), ws_bytes,
                                       _stream(stream)))


def head_logits(dt: int, B: int, hidden: int, vocab: int, n_heads: int, h, head_w, logits_out,
                head_layout: int = HEADS_ROWMAJOR, stream=None):
    _check(load().specmemo_head_logits(dt, B, hidden, vocab, n_heads, _ptr(h), _ptr(head_w), head_layout,
                                       _ptr(logits_out), _stream(stream)))


def medusa_resblock(dt: int, B: int, hidden: int, n_heads: int, h, w1, b1, out, w1_layout: int = HEADS_PACKED,
                    stream=None):
    _check(load().specmemo_medusa_resblock(dt, B, hidden, n_heads, _ptr(h), _ptr(w1), w1_layout, _ptr(b1),
                                           _ptr(out), _stream(stream)))


def sample_next(dt: int, trees: Trees, vocab: int, temperature: float, seed: int, offset: int, base_logits,
                accept_len, path, path_stride: int, next_tok, ws=None, ws_bytes: int = 0, stream=None):
    ts = trees.struct()
    _check(load().specmemo_sample_next(dt, C.byref(ts), vocab, temperature, seed, offset, _ptr(base_logits),
                                       _ptr(accept_len), _ptr(path), path_stride, _ptr(next_tok), _ptr(ws),
                                       ws_bytes, _stream(stream)))


def packed_heads_bytes(dt: int, n_heads: int, vocab: int, hidden: int) -> int:
    return int(load().specmemo_packed_heads_bytes(dt, n_heads, vocab, hidden))


def pack_heads(dt: int, n_heads: int, vocab: int, hidden: int, src, dst, stream=None):
    _check(load().specmemo_pack_heads(dt, n_heads, vocab, hidden, _ptr(src), _ptr(dst), _stream(stream)))


def tree_attn(dt: int, trees: Trees, kv: KVPool, n_q: int, q, out, scale: float = 0.0, ws=None,
              ws_bytes: int = 0, stream=None):
    ts, ks = trees.struct(), kv.struct()
    _check(load().specmemo_tree_attn(dt, C.byref(ts), C.byref(ks), n_q, scale, _ptr(q), _ptr(out), _ptr(ws),
                                     ws_bytes, _stream(stream)))


STATIC_SCRATCH_BYTES = 32 << 20


def tree_attn_noalloc(dt: int, trees: Trees, kv: KVPool, n_q: int, q, out, scale: float = 0.0, stream=None):
    ts, ks = trees.struct(), kv.struct()
    _check(load().specmemo_tree_attn_noalloc(dt, C.byref(ts), C.byref(ks), n_q, scale, _ptr(q), _ptr(out),
                                             _stream(stream)))


def accept(dt: int, trees: Trees, vocab: int, mode: int, base_logits, node_tok, accept_len, path, path_stride: int,
           next_tok, temperature: float = 1.0, eps: float = 0.09, delta: float = 0.3, ws=None, ws_bytes: int = 0,
           stream=None):
    ts = trees.struct()
    _check(load().specmemo_accept(dt, C.byref(ts), vocab, mode, temperature, eps, delta, _ptr(base_logits),
                                  _ptr(node_tok), _ptr(accept_len), _ptr(path), path_stride, _ptr(next_tok),
                                  _ptr(ws), ws_bytes, _stream(stream)))


def accept_compact(dt: int, trees: Trees, kv: KVPool, vocab: int, mode: int, base_logits, node_tok, accept_len, path,
                   path_stride: int, next_tok, temperature: float = 1.0, eps: float = 0.09, delta: float = 0.3,
                   ws=None, ws_bytes: int = 0, stream=None):
    ts, ks = trees.struct(), kv.struct()
    _check(load().specmemo_accept_compact(dt, C.byref(ts), C.byref(ks), vocab, mode, temperature, eps, delta,
                                          _ptr(base_logits), _ptr(node_tok), _ptr(accept_len), _ptr(path),
                                          path_stride, _ptr(next_tok), _ptr(ws), ws_bytes, _stream(stream)))


def kv_compact(dt: int, trees: Trees, kv: KVPool, accept_len, path, path_stride: int, stream=None):
    ts, ks = trees.struct(), kv.struct()
    _check(load().specmemo_kv_compact(dt, C.byref(ts), C.byref(ks), _ptr(accept_len), _ptr(path), path_stride,
                                      _stream(stream)))


# ---- padded batching -------------------------------------------------------------

def key_mask_words(cap_total: int) -> int:
    return int(load().specmemo_key_mask_words(cap_total))


def pack_key_valid(flags) -> np.ndarray:
    """Per-row flags (nonzero = token, 0 = pad) -> the library's uint32 words
    (bit r % 32 of word r / 32), padded to key_mask_words(len(flags))."""
    f = np.asarray(flags) != 0
    words = np.zeros(key_mask_words(len(f)), np.uint32)
    packed = np.packbits(f, bitorder="little")
    packed = np.concatenate([packed, np.zeros((-len(packed)) % 4, np.uint8)])
    words[:len(packed) // 4] = packed.view("<u4")
    return words


def unpack_key_valid(words, cap_total: int) -> np.ndarray:
    """Inverse of pack_key_valid: uint8 flags [cap_total]."""
    w = np.ascontiguousarray(np.asarray(words, dtype=np.uint32))
    return np.unpackbits(w.view(np.uint8), bitorder="little")[:cap_total]


def _words(key_valid, words):
    if words is not None:
        return words
    return int(key_valid.numel()) if hasattr(key_valid, "numel") else len(key_valid)


def tree_attn_padded(dt: int, trees: Trees, kv: KVPool, key_valid, n_q: int, q, out, scale: float = 0.0, ws=None,
                     ws_bytes: int = 0, stream=None, key_valid_words=None):
    ts, ks = trees.struct(), kv.struct()
    _check(load().specmemo_tree_attn_padded(dt, C.byref(ts), C.byref(ks), _ptr(key_valid),
                                            _words(key_valid, key_valid_words), n_q, scale, _ptr(q), _ptr(out),
                                            _ptr(ws), ws_bytes, _stream(stream)))


def kv_pad_update(dt: int, trees: Trees, kv: KVPool, accept_len, path, path_stride: int, key_valid, pos, ws=None,
                  ws_bytes: int = 0, stream=None, key_valid_words=None):
    ts, ks = trees.struct(), kv.struct()
    _check(load().specmemo_kv_pad_update(dt, C.byref(ts), C.byref(ks), _ptr(accept_len), _ptr(path), path_stride,
                                         _ptr(key_valid), _words(key_valid, key_valid_words), _ptr(pos), _ptr(ws),
                                         ws_bytes, _stream(stream)))


# ---- memory budget and tree construction (host) ------------------------------

def _bytes(v: int) -> int:
    if v < 0:
        raise SpecmemoError(-1, load().specmemo_last_error().decode())
    return int(v)


def mem_kv_bytes(layers: int, batch: int, n_kv: int, head_dim: int, tokens: int, elem_bytes: int) -> int:
    return _bytes(load().specmemo_mem_kv_bytes(layers, batch, n_kv, head_dim, tokens, elem_bytes))


def mem_buffer_bytes(batch: int, nodes: int, seqs: int, levels: int, vocab: int, elem_bytes: int) -> int:
    return _bytes(load().specmemo_mem_buffer_bytes(batch, nodes, seqs, levels, vocab, elem_bytes))


def mem_total_bytes(base_model_bytes: int, head_bytes: int, heads: int, kv: int, buffers: int) -> int:
    return _bytes(load().specmemo_mem_total_bytes(base_model_bytes, head_bytes, heads, kv, buffers))


def tree_full_nodes(arity: int, levels: int) -> int:
    return _bytes(load().specmemo_tree_full_nodes(arity, levels))


def tree_build(nodes: int, leaves: int, max_depth: int, arity: int):
    """(parent, depth, rank) int32 arrays of the built tree."""
    out = [np.zeros(max(nodes, 1), np.int32) for _ in range(3)]
    _check(load().specmemo_tree_build(nodes, leaves, max_depth, arity, *(a.ctypes.data for a in out)))
    return tuple(out)


def tree_leaves(parent, depth, rank) -> int:
    p, d, r = _i32(parent), _i32(depth), _i32(rank)
    s = load().specmemo_tree_leaves(len(p), p.ctypes.data, d.ctypes.data, r.ctypes.data)
    if s < 0:
        raise SpecmemoError(-3, load().specmemo_last_error().decode())
    return int(s)


def tree_prune(parent, depth, rank, keep: Sequence[int]):
    """Right-to-left pruning with per-level keep counts; (parent, depth, rank) of the kept nodes."""
    p, d, r, k = _i32(parent), _i32(depth), _i32(rank), _i32(keep)
    n = len(p)
    out = [np.zeros(max(n, 1), np.int32) for _ in range(3)]
    m = C.c_int32(0)
    _check(load().specmemo_tree_prune(n, p.ctypes.data, d.ctypes.data, r.ctypes.data, len(k),
                                      k.ctypes.data if len(k) else None, C.addressof(m),
                                      *(a.ctypes.data for a in out)))
    return tuple(a[:m.value].copy() for a in out)


def plan_budget(max_memory: int, base_model_bytes: int, head_bytes: int, layers: int, n_kv: int, head_dim: int,
                vocab: int, elem_bytes: int, batch: int, query_count: int, query_length: int, default_heads: int,
                default_tree) -> dict:
    """Alg. 1 without quantisation: dict(kind, heads, nodes, leaves, kv_bytes, total_bytes)."""
    parent, depth, rank = (_i32(a) for a in default_tree)
    m = _Budget(max_memory, base_model_bytes, head_bytes, layers, n_kv, head_dim, vocab, elem_bytes, batch,
                query_count, query_length, default_heads)
    out = _BudgetPlan()
    _check(load().specmemo_plan_budget(C.byref(m), len(parent), parent.ctypes.data, depth.ctypes.data,
                                       rank.ctypes.data, C.byref(out)))
    return {f: int(getattr(out, f)) for f, _ in _BudgetPlan._fields_}


def plan_tree_sizes(seq_len, seq_cap, default_nodes: int) -> np.ndarray:
    ln, cp = _i32(seq_len), _i32(seq_cap)
    out = np.zeros(max(len(ln), 1), np.int32)
    _check(load().specmemo_plan_tree_sizes(len(ln), ln.ctypes.data, cp.ctypes.data, default_nodes, out.ctypes.data))
    return out[:len(ln)]
