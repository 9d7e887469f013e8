"""The LDS-wait rule the kernels rely on, checked on a model of the wave's
LGKM counter (CPU only).

A wave's LDS operations complete in issue order; its scalar-memory loads
(s_load, s_memtime) share the same counter and may complete in any order
relative to them and to each other.  "s_waitcnt lgkmcnt(n)" blocks until at
most n counted operations are outstanding.  The kernels' signal() and the
generated consumer loop wait with n = the number of LDS operations issued
after the last one they need.  This test enumerates every issue sequence of
up to 6 LDS and 2 scalar operations and every completion order the rules
allow, and checks that whenever the wait is satisfied the needed LDS
operation has completed, whatever scalar loads are in flight; and that a
wait one weaker (n + 1) does not give that guarantee.
"""
import itertools


def completion_orders(ops):
    """All orders in which the issued ops may complete: LDS ops ('L', i) in
    issue order, scalar ops ('S', j) anywhere."""
    lds = [o for o in ops if o[0] == "L"]
    scal = [o for o in ops if o[0] == "S"]
    n = len(ops)
    for pos in itertools.permutations(range(n), len(scal)):
        order = [None] * n
        for p, s in zip(pos, scal):
            order[p] = s
        it = iter(lds)
        yield [o if o is not None else next(it) for o in order]


def wait_guarantees(ops, need, n):
    """True if lgkmcnt(n) being satisfied implies op `need` has completed, for
    every allowed completion order and every point in it."""
    for order in completion_orders(ops):
        done = set()
        for k in range(len(order) + 1):
            if k:
                done.add(order[k - 1])
            if len(ops) - len(done) <= n and need not in done:
                return False
    return True


def sequences(max_lds=6, max_scal=2):
    for nl in range(1, max_lds + 1):
        for ns in range(0, max_scal + 1):
            for spos in itertools.combinations(range(nl + ns), ns):
                ops, li, si = [], 0, 0
                for p in range(nl + ns):
                    if p in spos:
                        ops.append(("S", si))
                        si += 1
                    else:
                        ops.append(("L", li))
                        li += 1
                yield ops


def test_wait_on_younger_lds_count_is_safe_with_scalar_loads_in_flight():
    checked = 0
    for ops in sequences():
        lds = [o for o in ops if o[0] == "L"]
        for i, need in enumerate(lds):
            younger = len(lds) - 1 - i
            assert wait_guarantees(ops, need, younger), (ops, need, younger)
            checked += 1
    assert checked > 500


def test_one_weaker_wait_is_not_safe():
    for ops in sequences(max_lds=4, max_scal=1):
        lds = [o for o in ops if o[0] == "L"]
        for i, need in enumerate(lds):
            younger = len(lds) - 1 - i
            assert not wait_guarantees(ops, need, younger + 1), (ops, need)
