"""MI355X-native tree verification for Medusa-style speculative decoding (SpecMemo).

The hot path of one speculative step (SpecMemo, Sec. 3.1 and App. A.1):

  (a) Medusa-head projection of the last hidden state and per-head top-k,
      assembled into a fixed candidate tree,
  (b) tree-masked attention of every candidate node against its sequence's
      committed KV plus its own tree ancestors, over a ragged batch,
  (c) greedy or typical acceptance of the longest accepted root-to-leaf path,
  (d) in-place compaction of the accepted path's K/V inside a preallocated,
      budget-capped KV pool.

Each stage is a hand-written HIP kernel for gfx950 behind the C ABI declared
in ``include/specmemo.h``; ``specmemo`` is the ctypes binding.  Importing this
package loads nothing: the binding loads the shared library on first use and
raises if it was not built.
"""

__all__ = ["configs", "synth", "specmemo"]
