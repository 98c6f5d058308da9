"""The dependency cases of Section 5.2, decided from the loop tree.

TEST INFRASTRUCTURE ONLY: used by the tests to check the library's
classification; the GPU library never imports it.

For a dependency (p, c, k), S is the innermost loop enclosing both p and c
and P the loop whose body holds p directly.  Each instruction is placed in
S's body at the item (a block, or a loop nested in S) that contains it;
inside one block the listing order decides.  The dependency is forward when
c's place follows p's.  Section 5.2 allows:

  * C1, P = S: any offset, except that offset 0 needs p before c;
  * C2, P nested in S, forward: offset 0 only;
  * C3, P nested in S, backward: offset 1 only (offset 0 can never be met).

Every other nested offset falls back to the barrier scheme of Section 3.4:
a barrier at the end of every iteration of S orders all instances of an
earlier iteration of S, which is all the dependency asks for when k >= 1.
With S the top-level loop (one iteration) such a dependency is never owed.
"""
from __future__ import annotations

ORDER = "order"        # offset 0 with the consumer not after the producer
NOT_ALLOCATABLE = "not allocatable"
C1, C2, C3, FALLBACK = 1, 2, 3, 4
LINEAR = 6             # extension, not in the paper: offset counted across trips of S


def _home(prog):
    """Innermost loop of every instruction, and the (item, listing) place of
    every instruction within that loop's body."""
    home, place = {}, {}
    for l, items in enumerate(prog.body):
        for j, (kind, bid) in enumerate(items):
            if kind == 0:
                for pos, i in enumerate(prog.blocks[bid]):
                    home[i] = l
                    place[i] = (j, pos)
    return home, place


def _chain(prog, l):
    """Loops from l up to the top level, l first."""
    out = [l]
    while prog.loop_parent[out[-1]] >= 0:
        out.append(prog.loop_parent[out[-1]])
    return out


def _item_of_loop(prog, child, S):
    """Index in S's body of the item that is, or contains, loop ``child``."""
    while prog.loop_parent[child] != S:
        child = prog.loop_parent[child]
    for j, (kind, bid) in enumerate(prog.body[S]):
        if kind == 1 and bid == child:
            return j
    raise ValueError("loop not in its parent's body")


def classify(prog, d):
    """(case, S, P, forward) of dependency d; case is C1, C2, C3, FALLBACK,
    ORDER, or for a dependency flagged linearized LINEAR or
    NOT_ALLOCATABLE."""
    p, c, k = prog.deps[d]
    home, place = _home(prog)
    P = home[p]
    cp, cc = _chain(prog, P), _chain(prog, home[c])
    S = next(l for l in cp if l in cc)

    def where(i):
        if home[i] == S:
            return place[i]
        return (_item_of_loop(prog, home[i], S), -1)

    forward = where(p) < where(c)
    if getattr(prog, "dep_linear", None) and prog.dep_linear[d]:
        # the linearized reading of the offset (an extension): only for a
        # producer directly in S, whose count of S is then its own count
        if P != S:
            return NOT_ALLOCATABLE, S, P, forward
        return (ORDER if (not forward and k == 0) else LINEAR), S, P, forward
    if P == S:
        case = C1 if (forward or k >= 1) else ORDER
    elif forward:
        case = C2 if k == 0 else FALLBACK
    else:
        case = ORDER if k == 0 else (C3 if k == 1 else FALLBACK)
    return case, S, P, forward


def barrier_loops(prog):
    """Loops whose every iteration end carries a fallback barrier."""
    out = set()
    for d in range(len(prog.deps)):
        case, S, _, _ = classify(prog, d)
        if case == FALLBACK and S != 0:
            out.add(S)
    return out
