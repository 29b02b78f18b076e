"""The LDS tile ring of tree_attn_bf16, checked as a protocol on the CPU.

The kernel stages 64-key K and V tiles in SLOTS-deep rings filled by direct
global->LDS loads that complete in issue order per wave (vmcnt), waits on
them with explicit vmcnt counts, and separates reuse of a slot from reads of
its previous tile with a bare workgroup barrier (after lgkmcnt(0), so a wave's
own LDS reads are done when it arrives).  The tree's parent array is written
into the last V slot before the prologue barrier and read (the ancestor walk)
between that barrier and the first loop barrier.

`kernel_program` writes down, per wave, the order of those events in the
kernel (every wave runs the same order); `check` proves, for every batch of
tiles, that under any completion times the hardware may choose:

* a read of tile j in a slot happens after every wave's loads of tile j into
  that slot have been forced complete before a barrier the reader has passed;
* a load into a slot is issued only after every wave's last read of the
  slot's previous content (no write can land under a read);
* no load is still in flight when the program ends;
* the parent array is not overwritten before the ancestor walk is done.

The key-split form (two key groups per row block) then writes its second
group's (m, l, O) over the rings for the first group to merge: that needs
every load complete and every wave's reads behind a barrier.

The mutants at the bottom show that the checker rejects the plausible ways
to get the ring wrong (a wait one tile too shallow, a load issued before the
barrier, a third slot without the deeper wait count, the parent array in a
slot the prologue fills, the merge without its barrier).
"""

import itertools

import pytest


def kernel_program(ntiles, slots, *, par_slot=None, wait_later=None, issue_before_barrier=False, merge=False,
                   merge_barrier=True):
    """Event list of one wave.  Events: ("issue", tile, op), ("wait", k),
    ("barrier",), ("read", tile, op), ("par_write",), ("par_read",), ("merge",).
    `merge`: the key-split form, whose two key groups exchange (m, l, O)
    through the K and V rings after the loop, behind one more barrier."""
    par_slot = slots - 1 if par_slot is None else par_slot
    if wait_later is None:
        def wait_later(j):
            # loads issued after tile j's: tile j+1 (K and V) with three slots
            return 2 if (slots == 3 and j + 1 < ntiles) else 0
    ev = [("par_slot", par_slot)]
    for t in range(slots - 1):                 # prologue: tiles 0 .. SLOTS-2
        if t < ntiles:
            ev += [("issue", t, "K"), ("issue", t, "V")]
    # The Q fragments are loaded after the tiles and landed before the loop;
    # the model does not rely on that wait (the loop's waits must suffice).
    ev += [("par_write",), ("barrier",), ("par_read",)]
    for j in range(ntiles):
        ev.append(("wait", wait_later(j)))
        nxt = j + slots - 1
        if issue_before_barrier and nxt < ntiles:
            ev += [("issue", nxt, "K"), ("issue", nxt, "V")]
        ev.append(("barrier",))
        if not issue_before_barrier and nxt < ntiles:
            ev += [("issue", nxt, "K"), ("issue", nxt, "V")]
        ev += [("read", j, "K"), ("read", j, "V")]
    if merge:
        ev += ([("barrier",)] if merge_barrier else []) + [("merge",)]
    return ev


def check(ev, slots):
    """Raise AssertionError on the first protocol violation of the program
    `ev` (run by every wave of the block)."""
    par_slot = ev[0][1]
    epoch = 0                 # barriers passed
    issued = []               # (tile, op, epoch issued) in issue order
    done_by = {}              # load index -> epoch before whose barrier it is forced complete
    pending = []              # indices of loads not yet forced complete
    reads = []                # (epoch, slot key, tile)
    for e in ev[1:]:
        kind = e[0]
        if kind == "issue":
            _, t, op = e
            issued.append((t, op, epoch))
            pending.append(len(issued) - 1)
        elif kind == "wait":
            k = e[1]
            keep = pending[len(pending) - k:] if k else []
            for i in pending[:len(pending) - k] if k else pending:
                done_by[i] = epoch     # complete before this wave's next barrier
            pending = keep
        elif kind == "barrier":
            epoch += 1
        elif kind == "read":
            _, t, op = e
            reads.append((epoch, (op, t % slots), t))
            # every wave's loads of (t, op) were issued and forced complete before
            # a barrier this read follows; all waves run the same program, so
            # "before barrier number epoch" in this program is the condition
            for i, (tt, oo, ep) in enumerate(issued):
                if (tt, oo) == (t, op):
                    assert i in done_by and done_by[i] < epoch, f"read of {op}{t} before its load is complete"
            assert any((tt, oo) == (t, op) for tt, oo, _ in issued), f"read of {op}{t} never loaded"
        elif kind == "par_write":
            reads.append((epoch, ("V", par_slot), -1))   # an LDS write: no load may land under it either
        elif kind == "par_read":
            reads.append((epoch, ("V", par_slot), -1))
        elif kind == "merge":
            # LDS writes over both rings: no load may still be landing, and
            # every wave's reads of the rings must be behind a barrier
            assert not pending, "merge writes while a tile load is in flight"
            assert all(re < epoch for (re, _, _) in reads), "merge writes over a ring another wave may still read"
        else:
            raise ValueError(kind)
    assert not pending, "loads still in flight at the end of the program"
    # A load into a slot may write from its issue (epoch e, after barrier e)
    # until it is complete.  Any read of another content of that slot in
    # epoch >= e by any wave could overlap it; reads in earlier epochs ended
    # before their wave arrived at barrier e (lgkmcnt(0)).
    for (t, op, e) in issued:
        key = (op, t % slots)
        for (re, rkey, rt) in reads:
            if rkey == key and rt != t and re >= e:
                # the slot's earlier content is read at or after the issue
                assert rt > t, f"load of {op}{t} issued in epoch {e} while {op}{rt} in the slot is read in epoch {re}"
                # a later tile's read is fine only if it follows this load's completion
                # (checked above) and the later tile's own issue (below)
    # And a slot's content must be read only while it is that content: between
    # the completion of its load and the issue of the next load into the slot.
    for (re, key, rt) in reads:
        if rt < 0:
            continue
        nxt = [e for (t, op, e) in issued if (op, t % slots) == key and t > rt]
        if nxt:
            assert re < min(nxt), f"{key[0]}{rt} read in epoch {re} after the slot's next load was issued"


CASES = [(n, s) for s in (2, 3) for n in range(1, 9)]


@pytest.mark.parametrize("ntiles,slots", CASES)
def test_ring_protocol_of_the_kernel(ntiles, slots):
    check(kernel_program(ntiles, slots), slots)


@pytest.mark.parametrize("ntiles", range(1, 9))
def test_ring_protocol_with_key_split_merge(ntiles):
    check(kernel_program(ntiles, 2, merge=True), 2)


def test_mutant_merge_without_barrier_is_caught():
    for n in range(1, 6):
        with pytest.raises(AssertionError):
            check(kernel_program(n, 2, merge=True, merge_barrier=False), 2)


def test_mutant_wait_too_shallow_is_caught():
    # two slots but waiting as if tile j+1 could stay in flight
    for n in range(2, 6):
        with pytest.raises(AssertionError):
            check(kernel_program(n, 2, wait_later=lambda j: 2 if j + 1 < n else 0), 2)


def test_mutant_issue_before_barrier_is_caught():
    for n, s in itertools.product(range(2, 6), (2, 3)):
        if n >= s:
            with pytest.raises(AssertionError):
                check(kernel_program(n, s, issue_before_barrier=True), s)


def test_mutant_three_slot_wait_counts():
    # with three slots, waiting for everything is merely slower (still safe) ...
    for n in range(1, 7):
        check(kernel_program(n, 3, wait_later=lambda j: 0), 3)
    # ... while allowing tile j itself to stay in flight is caught
    for n in range(1, 7):
        with pytest.raises(AssertionError):
            check(kernel_program(n, 3, wait_later=lambda j: 4 if j + 1 < n else 2), 3)


def test_mutant_parent_array_in_a_prologue_slot_is_caught():
    for s in (2, 3):
        with pytest.raises(AssertionError):
            check(kernel_program(4, s, par_slot=0), s)
