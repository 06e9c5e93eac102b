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
