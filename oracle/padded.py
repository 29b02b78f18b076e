"""Padded batching of SpecMemo (Sec. 3.3, Fig. 8).  TEST INFRASTRUCTURE.

Plain Python over host copies of the KV pool.  The paper keeps a batch's
tensors uniform by padding: after verification every sequence's accepted
tokens are padded to the batch's longest acceptance, the pad tokens stay in
the cache and are masked with -inf in later attention, and position IDs skip
them.  Only the tests may import this module; it shares nothing with the
library.

Readings: a sequence commits tau_b = accept_len[b] + 1 tokens (the root and
its accepted descendants); the uniform length is T = max_b tau_b; the accepted
rows move to slab rows L_b .. L_b + tau_b - 1 as in compaction; rows
L_b + tau_b .. L_b + T - 1 are pad tokens (their contents are whatever the
tree left there); every sequence's cache grows by T rows and its position by
tau_b.  Only committed rows can be pads: this step's tree rows never are.
"""

from __future__ import annotations

import numpy as np

from . import kv_compact


def pad_update(K, V, seq_base, seq_len, pos, key_valid, accept_len, path):
    """One padded bookkeeping step on host copies (K, V, key_valid modified in
    place).  Returns (new seq_len, new pos)."""
    acc = np.asarray(accept_len, dtype=np.int64)
    L = np.asarray(seq_len, dtype=np.int64)
    kv_compact(K, V, seq_base, seq_len, accept_len, path)      # the accepted rows, in order
    tau = acc + 1
    T = int(tau.max()) if len(tau) else 0
    for b in range(len(tau)):
        first = int(seq_base[b]) + int(L[b])
        for j in range(T):
            key_valid[first + j] = 1 if j < tau[b] else 0     # a pad token past the acceptance
    new_len = (L + T).astype(np.int32)
    new_pos = (np.asarray(pos, dtype=np.int64) + tau).astype(np.int32)
    return new_len, new_pos
