"""Exhaustive check of the split-K arrival protocol on a model (CPU).

The kernel's protocol for the K slices of one tile, as steps of one
workgroup (the persistent grid gives workgroup g the units g, g+G, ...;
unit u is slice u % S of tile u // S):

  ticket = cnt[t]++                       (relaxed add)
  if ticket < S-1:  write partial[t][s];  written[t]++ ; next unit
  else:             wait written[t] >= S-1; read every other partial;
                    cnt[t] = written[t] = 0 ; epilogue ; next unit

The model runs every interleaving of these steps with at most R workgroups
resident at once (a workgroup becomes resident only when a slot is free and
leaves it when its units are done), R down to 1, so no co-residency is
assumed.  In every reachable state some resident workgroup can move (no
deadlock), each tile is reduced exactly once, the reducer finds every other
slice's partial written, and the counters end at zero.
"""
from __future__ import annotations

from functools import lru_cache

import pytest

# program counter of a workgroup inside its current unit
START, WRITE, COUNT, WAIT, READ, RESET, DONE = range(7)


def _explore(T: int, S: int, G: int, R: int, wait_target: int | None = None) -> int:
    target = S - 1 if wait_target is None else wait_target
    units = [[u for u in range(g, T * S, G)] for g in range(G)]

    @lru_cache(maxsize=None)
    def reachable(state) -> int:
        # state: (per-wg (unit index, pc, ticket), resident tuple, cnt, written,
        #         partials bitmask per tile, reduced count per tile)
        wgs, resident, cnt, written, parts, reduced = state
        if all(i == len(units[g]) for g, (i, _, _) in enumerate(wgs)):
            assert all(c == 0 for c in cnt) and all(w == 0 for w in written), "counters left"
            assert all(r == 1 for r in reduced), f"tiles reduced {reduced}"
            return 1
        moves = []
        # a waiting workgroup may become resident when a slot is free
        if len(resident) < R:
            for g in range(G):
                if g not in resident and wgs[g][0] == 0 and wgs[g][1] == START and units[g]:
                    moves.append(("admit", g))
        for g in resident:
            i, pc, ticket = wgs[g]
            u = units[g][i]
            t, s = divmod(u, S)
            if pc == WAIT and written[t] < target:
                continue                                   # blocked
            moves.append(("step", g))
        assert moves, f"deadlock in {state}"
        total = 0
        for kind, g in moves:
            w, res = list(wgs), list(resident)
            c, wr, pa, rd = list(cnt), list(written), list(parts), list(reduced)
            if kind == "admit":
                res.append(g)
                total += reachable((tuple(w), tuple(res), tuple(c), tuple(wr), tuple(pa),
                                    tuple(rd)))
                continue
            i, pc, ticket = w[g]
            t, s = divmod(units[g][i], S)
            if pc == START:                                # take a ticket
                ticket = c[t]
                c[t] += 1
                pc = WRITE if ticket < S - 1 else WAIT
            elif pc == WRITE:                              # write this slice's partial
                pa[t] |= 1 << s
                pc = COUNT
            elif pc == COUNT:                              # count it (after the release)
                wr[t] += 1
                pc = DONE
            elif pc == WAIT:                               # the others have counted
                pc = READ
            elif pc == READ:                               # acquire and read the others
                others = ((1 << S) - 1) & ~(1 << s)
                assert pa[t] & others == others, "reducer read an unwritten partial"
                pc = RESET
            elif pc == RESET:
                c[t] = wr[t] = 0
                rd[t] += 1
                pc = DONE
            if pc == DONE:
                i, pc, ticket = i + 1, START, 0
                if i == len(units[g]):
                    res.remove(g)                          # leaves its slot
            w[g] = (i, pc, ticket)
            total += reachable((tuple(w), tuple(res), tuple(c), tuple(wr), tuple(pa), tuple(rd)))
        return total

    init = (tuple((0, START, 0) for _ in range(G)), (), (0,) * T, (0,) * T, (0,) * T, (0,) * T)
    n = reachable(init)
    reachable.cache_clear()
    return n


@pytest.mark.parametrize("T,S,G,R", [
    (1, 2, 2, 2), (1, 2, 2, 1),          # two slices, both resident / one at a time
    (1, 3, 3, 1), (1, 3, 2, 1),          # a workgroup holds two slices of one tile
    (2, 2, 3, 2), (2, 3, 2, 2),          # slices of two tiles spread over the grid
    (2, 2, 4, 1), (1, 4, 4, 2),
])
def test_split_k_protocol_never_deadlocks_and_reduces_once(T, S, G, R):
    assert _explore(T, S, G, R) >= 1


def test_model_finds_a_planted_protocol_error():
    """Pin of the model itself: a reducer that waits until all S slices have
    counted (itself included, which never counts) can never proceed, and the
    explorer reports the deadlock."""
    with pytest.raises(AssertionError, match="deadlock"):
        _explore(1, 2, 2, 2, wait_target=2)
    with pytest.raises(AssertionError, match="deadlock"):
        _explore(2, 3, 2, 1, wait_target=3)
    # and a reducer that does not wait breaks the other invariants: it reads
    # a partial before it is written, or resets a counter its partner then
    # increments (whichever interleaving the search reaches first)
    with pytest.raises(AssertionError, match="unwritten partial|counters left"):
        _explore(1, 2, 2, 2, wait_target=0)


# ---------------------------------------------------------------------------
# Timeouts.  A reducer whose bounded wait expires records ETIMEOUT and gives
# the tile up without resetting its counters, because slices of that call
# that already hold a ticket may still count themselves afterwards.  A later
# call on the same workspace then draws tickets at or past S for that tile,
# and each such slice reports a stale workspace and skips the tile instead
# of taking part (and instead of a reducer summing partials that were never
# written in that call).

def _run_call(T, S, G, R, cnt0, written0, allow_timeout, reset_on_timeout, check_tickets):
    """Every interleaving of one call starting from counters cnt0/written0.
    Returns the set of end states (cnt, written, reduced, flagged, timed_out)."""
    units = [[u for u in range(g, T * S, G)] for g in range(G)]
    ends = set()
    seen = set()

    def explore(state):
        if state in seen:
            return
        seen.add(state)
        wgs, resident, cnt, written, parts, reduced, flagged, timed = state
        if all(i == len(units[g]) for g, (i, _, _) in enumerate(wgs)):
            ends.add((cnt, written, reduced, flagged, timed))
            return
        moves = []
        if len(resident) < R:
            for g in range(G):
                if g not in resident and wgs[g][0] == 0 and wgs[g][1] == START and units[g]:
                    moves.append(("admit", g))
        for g in resident:
            i, pc, _ = wgs[g]
            t, _s = divmod(units[g][i], S)
            if pc == WAIT and written[t] < S - 1:
                if allow_timeout:
                    moves.append(("timeout", g))
                continue
            moves.append(("step", g))
        assert moves, f"deadlock in {state}"
        for kind, g in moves:
            w, res = list(wgs), list(resident)
            c, wr, pa = list(cnt), list(written), list(parts)
            rd, fl, tm = list(reduced), list(flagged), list(timed)
            if kind == "admit":
                res.append(g)
                explore((tuple(w), tuple(res), tuple(c), tuple(wr), tuple(pa), tuple(rd),
                         tuple(fl), tuple(tm)))
                continue
            i, pc, ticket = w[g]
            t, s = divmod(units[g][i], S)
            if kind == "timeout":
                tm[t] += 1
                if reset_on_timeout:
                    c[t] = wr[t] = 0
                pc = DONE
            elif pc == START:
                ticket = c[t]
                c[t] += 1
                if check_tickets and ticket >= S:
                    fl[t] += 1                             # stale workspace: skip the tile
                    pc = DONE
                else:
                    pc = WAIT if ticket + 1 == S else WRITE
            elif pc == WRITE:
                pa[t] |= 1 << s
                pc = COUNT
            elif pc == COUNT:
                wr[t] += 1
                pc = DONE
            elif pc == WAIT:
                pc = READ
            elif pc == READ:
                others = ((1 << S) - 1) & ~(1 << s)
                assert pa[t] & others == others, "reducer read an unwritten partial"
                pc = RESET
            elif pc == RESET:
                c[t] = wr[t] = 0
                rd[t] += 1
                pc = DONE
            if pc == DONE:
                i, pc, ticket = i + 1, START, 0
                if i == len(units[g]):
                    res.remove(g)
            w[g] = (i, pc, ticket)
            explore((tuple(w), tuple(res), tuple(c), tuple(wr), tuple(pa), tuple(rd),
                     tuple(fl), tuple(tm)))

    explore((tuple((0, START, 0) for _ in range(G)), (), tuple(cnt0), tuple(written0),
             (0,) * T, (0,) * T, (0,) * T, (0,) * T))
    return ends


def _timeout_then_next_call(T, S, G, R, reset_on_timeout=False, check_tickets=True):
    zero = (0,) * T
    first = _run_call(T, S, G, R, zero, zero, True, reset_on_timeout, check_tickets)
    assert any(any(tm) for *_, tm in first), "the model never timed out"
    for cnt, written, reduced, flagged, timed in first:
        for t in range(T):
            # each tile of the first call is reduced once, or given up by a timeout
            assert reduced[t] + timed[t] == 1 and flagged[t] == 0, (reduced, timed)
        second = _run_call(T, S, G, R, cnt, written, False, reset_on_timeout, check_tickets)
        for _, _, reduced2, flagged2, _ in second:
            for t in range(T):
                clean = cnt[t] == 0 and written[t] == 0
                if clean:
                    assert reduced2[t] == 1 and flagged2[t] == 0, "clean tile not reduced once"
                else:
                    # every slice reports the stale workspace; nothing is summed
                    assert reduced2[t] == 0 and flagged2[t] == S, \
                        f"stale tile neither reduced nor reported ({reduced2}, {flagged2})"


@pytest.mark.parametrize("T,S,G,R", [(1, 2, 2, 2), (1, 3, 3, 2), (2, 2, 2, 2), (2, 2, 4, 2)])
def test_split_k_timeout_leaves_counters_and_the_next_call_reports_them(T, S, G, R):
    _timeout_then_next_call(T, S, G, R)


def test_timeout_model_finds_the_planted_errors():
    """Pins of the timeout model: resetting the counters on the timeout path
    lets a late arrival's count survive into the next call, whose reducer then
    passes its wait before its partner's partial is written; without the
    ticket check a stale tile is silently never written."""
    with pytest.raises(AssertionError, match="unwritten partial"):
        _timeout_then_next_call(1, 2, 2, 2, reset_on_timeout=True)
    with pytest.raises(AssertionError, match="neither reduced nor reported"):
        _timeout_then_next_call(1, 2, 2, 2, check_tickets=False)


# ---------------------------------------------------------------------------
# Banded reduction.  With one resident workgroup per slice, the tile's rows
# form S bands and every slice reduces and stores one of them:
#
#   ticket = cnt[t]++                     (ticket >= S: stale workspace, skip)
#   write the partial rows of the other bands ; written[t]++   (after a release)
#   wait written[t] >= S ; read the other slices' partials of band s
#   store band s ; u = cnt[t]++           (after a release)
#   if u == 2S-1: acquire, cnt[t] = written[t] = 0, publish the tile's counters
#
# Every slice waits for all the others, so the protocol needs them resident
# together; the host chooses it only when every unit has a workgroup of its
# own and the grid fits on the device at once.

B_START, B_WRITE, B_COUNT, B_WAIT, B_READ, B_STORE, B_TICKET2, B_PUBLISH, B_DONE = range(9)


def _explore_banded(T: int, S: int, R: int, wait_target: int | None = None,
                    publish_ticket: int | None = None) -> int:
    """Every interleaving of T tiles x S slices, one workgroup per slice, at
    most R resident at once.  Returns the number of terminal paths."""
    target = S if wait_target is None else wait_target
    last = 2 * S - 1 if publish_ticket is None else publish_ticket
    G = T * S
    full = (1 << S) - 1

    @lru_cache(maxsize=None)
    def reachable(state) -> int:
        pcs, resident, cnt, written, parts, stored, published = state
        if all(pc == B_DONE for pc in pcs):
            assert all(c == 0 for c in cnt) and all(w == 0 for w in written), "counters left"
            assert all(p == 1 for p in published), f"tiles published {published}"
            return 1
        moves = []
        if len(resident) < R:
            for g in range(G):
                if g not in resident and pcs[g] == B_START:
                    moves.append(("admit", g))
        for g in resident:
            t = g // S
            if pcs[g] == B_WAIT and written[t] < target:
                continue
            moves.append(("step", g))
        assert moves, f"deadlock in {state}"
        total = 0
        for kind, g in moves:
            pc, res = list(pcs), list(resident)
            c, wr, pa, st, pb = list(cnt), list(written), list(parts), list(stored), list(published)
            if kind == "admit":
                res.append(g)
            else:
                t, s = divmod(g, S)
                p = pc[g]
                if p == B_START:
                    ticket = c[t]
                    c[t] += 1
                    assert ticket < S, "first-round ticket past the slice count"
                    pc[g] = B_WRITE
                elif p == B_WRITE:
                    pa[t] |= 1 << s
                    pc[g] = B_COUNT
                elif p == B_COUNT:
                    wr[t] += 1
                    pc[g] = B_WAIT
                elif p == B_WAIT:
                    pc[g] = B_READ
                elif p == B_READ:
                    assert pa[t] == full, "a band summed before every partial was written"
                    pc[g] = B_STORE
                elif p == B_STORE:
                    st[t] |= 1 << s
                    pc[g] = B_TICKET2
                elif p == B_TICKET2:
                    u = c[t]
                    c[t] += 1
                    pc[g] = B_PUBLISH if u == last else B_DONE
                elif p == B_PUBLISH:
                    assert st[t] == full, "tile published before every band was stored"
                    c[t] = wr[t] = 0
                    pb[t] += 1
                    pc[g] = B_DONE
                if pc[g] == B_DONE:
                    res.remove(g)
            total += reachable((tuple(pc), tuple(res), tuple(c), tuple(wr), tuple(pa),
                                tuple(st), tuple(pb)))
        return total

    init = ((B_START,) * G, (), (0,) * T, (0,) * T, (0,) * T, (0,) * T, (0,) * T)
    n = reachable(init)
    reachable.cache_clear()
    return n


@pytest.mark.parametrize("T,S", [(1, 2), (1, 3), (1, 4), (2, 2)])
def test_banded_protocol_all_resident_publishes_once(T, S):
    assert _explore_banded(T, S, R=T * S) >= 1


def test_banded_model_finds_the_planted_errors():
    """Pins of the banded model: without co-residency it deadlocks (which is
    why the host requires one resident workgroup per slice); waiting for S-1
    counts lets a slice sum a band before the last partial is written;
    publishing on the second-to-last ticket publishes a tile with a band
    missing."""
    with pytest.raises(AssertionError, match="deadlock"):
        _explore_banded(1, 2, R=1)
    with pytest.raises(AssertionError, match="deadlock"):
        _explore_banded(1, 3, R=2)
    with pytest.raises(AssertionError, match="before every partial"):
        _explore_banded(1, 2, R=2, wait_target=1)
    with pytest.raises(AssertionError, match="before every band|counters left|published"):
        _explore_banded(1, 2, R=2, publish_ticket=2)


# ---------------------------------------------------------------------------
# Reduction kernel.  The first kernel's slices write their whole partials and
# take no ticket; the kernel boundary orders every partial before the second
# kernel, whose work units are (tile t, band b) of NB bands, on a persistent
# grid of G workgroups (workgroup g takes units g, g+G, ...):
#
#   c1 = written[t]                         (read before the sums; this mode
#                                            never changes written[])
#   sum band b of every partial ; store band b
#   u = cnt[t]++                            (after a release)
#   if c1 != 0 or u >= NB: report a stale workspace, publish nothing
#   elif u == NB-1: acquire, cnt[t] = 0, publish the tile's counters
#
# Nothing waits, so any grid and any number of resident workgroups work.

K_START, K_STORE, K_TICKET, K_PUBLISH, K_DONE = range(5)


def _run_reduction_kernel(T, NB, G, R, cnt0, written0, check_c1=True):
    """Every interleaving of the second kernel from counters cnt0/written0.
    Returns the set of end states (cnt, written, published, flagged)."""
    units = [[u for u in range(g, T * NB, G)] for g in range(G)]
    full = (1 << NB) - 1
    ends = set()
    seen = set()

    def explore(state):
        if state in seen:
            return
        seen.add(state)
        wgs, resident, cnt, stored, published, flagged = state
        if all(i == len(units[g]) for g, (i, _, _) in enumerate(wgs)):
            ends.add((cnt, tuple(written0), published, flagged))
            return
        moves = []
        if len(resident) < R:
            for g in range(G):
                if g not in resident and wgs[g][0] == 0 and wgs[g][1] == K_START and units[g]:
                    moves.append(("admit", g))
        moves += [("step", g) for g in resident]
        assert moves, f"deadlock in {state}"
        for kind, g in moves:
            w, res = list(wgs), list(resident)
            c, st, pb, fl = list(cnt), list(stored), list(published), list(flagged)
            if kind == "admit":
                res.append(g)
            else:
                i, pc, c1 = w[g]
                t, b = divmod(units[g][i], NB)
                if pc == K_START:
                    c1 = written0[t]
                    pc = K_STORE
                elif pc == K_STORE:
                    st[t] |= 1 << b
                    pc = K_TICKET
                elif pc == K_TICKET:
                    u = c[t]
                    c[t] += 1
                    stale = (check_c1 and c1 != 0) or u >= NB
                    if stale:
                        fl[t] += 1
                        pc = K_DONE
                    else:
                        pc = K_PUBLISH if u == NB - 1 else K_DONE
                elif pc == K_PUBLISH:
                    assert st[t] == full, "tile published before every band was stored"
                    c[t] = 0
                    pb[t] += 1
                    pc = K_DONE
                if pc == K_DONE:
                    i, pc, c1 = i + 1, K_START, 0
                    if i == len(units[g]):
                        res.remove(g)
                w[g] = (i, pc, c1)
            explore((tuple(w), tuple(res), tuple(c), tuple(st), tuple(pb), tuple(fl)))

    explore((tuple((0, K_START, 0) for _ in range(G)), (), tuple(cnt0), (0,) * T, (0,) * T,
             (0,) * T))
    return ends


@pytest.mark.parametrize("T,NB,G,R", [(1, 2, 2, 2), (1, 4, 4, 4), (1, 4, 1, 1), (2, 2, 3, 1),
                                      (2, 3, 4, 2), (3, 2, 6, 6)])
def test_reduction_kernel_publishes_each_tile_once_on_any_grid(T, NB, G, R):
    """From clean counters: each tile published exactly once, only after all
    its bands are stored, nothing reported, the ticket counter back at zero,
    whatever the grid and however few workgroups are resident."""
    zero = (0,) * T
    for cnt, written, published, flagged in _run_reduction_kernel(T, NB, G, R, zero, zero):
        assert cnt == zero and written == zero
        assert published == (1,) * T and flagged == zero


@pytest.mark.parametrize("T,S,G,R,NB", [(1, 2, 2, 2, 2), (1, 2, 2, 2, 4), (1, 3, 3, 2, 4),
                                        (2, 2, 2, 2, 2)])
def test_reduction_kernel_after_a_timeout_publishes_no_stale_tile(T, S, G, R, NB):
    """Counters left by a timed-out last-slice call (every end state of the
    timeout model): a tile whose ticket counter is non-zero always has a
    non-zero written counter too, which is what the reduction kernel reads;
    such a tile is reported by every band and never published, and its
    counters stay non-zero, so later calls report it as well; clean tiles are
    published once."""
    zero = (0,) * T
    first = _run_call(T, S, G, R, zero, zero, True, False, True)
    assert any(any(tm) for *_, tm in first), "the model never timed out"
    for cnt, written, *_ in first:
        for t in range(T):
            assert cnt[t] == 0 or written[t] != 0, (cnt, written)
        for cnt2, written2, published, flagged in _run_reduction_kernel(T, NB, NB, NB, cnt,
                                                                         written):
            for t in range(T):
                if cnt[t] == 0 and written[t] == 0:
                    assert published[t] == 1 and flagged[t] == 0 and cnt2[t] == 0
                else:
                    assert published[t] == 0 and flagged[t] == NB, (published, flagged)
                    assert cnt2[t] != 0 or written2[t] != 0


def test_reduction_kernel_model_finds_the_planted_error():
    """Pin: with the ticket check alone (no read of the written counter), a
    tile left with S < NB tickets by a timed-out call is published after only
    NB - S of its bands are stored."""
    with pytest.raises(AssertionError, match="before every band"):
        _run_reduction_kernel(1, 4, 4, 4, (2,), (1,), check_c1=False)
