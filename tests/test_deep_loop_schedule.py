"""Static check of the hand-placed LDS waits in the generated deep-prefetch K
loop (paper_2506_11209_amd/csrc/ws_deep_loop.inc).

The asm text of every configuration is interpreted along each path a tile
can take (no loop body up to five; each slot's counter found full at the
first look, after one poll, or after a failed poll) under the most pessimistic timing a
wave allows: an LDS operation completes only when a later s_waitcnt forces it
(operations complete in order, so lgkmcnt(n) completes all but the n most
recent).  Along every path:

  * each MFMA reads only fragment registers whose reads have completed;
  * each counter value is read (v_readfirstlane) only after its load completed;
  * a slot is released (ds_add to its empty counter) only after every read
    of that slot has completed;
  * no read is outstanding when the block ends, since the compiler may reuse
    the fragment registers afterwards;
  * every read stays inside its slot and the set it fills.

A wait that is one too weak anywhere fails one of these.  The file itself must
be what the generator writes."""
import os
import re
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2506_11209_amd", "csrc")
sys.path.insert(0, CSRC)
import gen_deep_loop as gen  # noqa: E402


def blocks():
    """{(tm, tn, tk, nc, split, bf16): [asm lines]} from the committed file."""
    with open(gen.OUT) as f:
        text = f.read()
    out = {}
    for m in re.finditer(r"struct DeepLoop<(\d+), (\d+), (\d+), (\d+), (\d+), (true|false)> \{(.*?)\n\};", text,
                         re.S):
        key = tuple(int(x) for x in m.groups()[:5]) + (m.group(6) == "true",)
        lines = re.findall(r'^\s*"(.*)\\n\\t"$', m.group(7), re.M)
        out[key] = [l.strip() for l in lines]
    return out


def regs(tok):
    m = re.fullmatch(r"v\[(\d+):(\d+)\]", tok)
    if m:
        return set(range(int(m.group(1)), int(m.group(2)) + 1))
    return {tok}  # a named operand such as %[vp]


class Sim:
    """One path through the block, with LDS operations completing only when
    a wait forces them.  K-iterations are numbered from the tile's first."""

    def __init__(self, cfg, iters, polls):
        self.c, self.iters, self.polls = cfg, iters, polls
        self.released = []
        self.pending = []  # [(registers written, K-iteration tag, description)] oldest first
        self.q = {"rs": None, "rb": None, "rel": None, "va": None, "vb": None, "slot": None}
        self.kss_a = None  # k-step of the A address in va (its XOR)
        self.kk = None
        self.errors = []

    def fail(self, msg):
        self.errors.append(msg)

    def wait(self, n):
        self.pending = self.pending[len(self.pending) - n:] if n else []

    def need(self, rs, what):
        for w, _, d in self.pending:
            if w & rs:
                self.fail("%s uses %s before its load (%s) completed" % (what, sorted(w & rs), d))

    def run(self, lines):
        labels = {}
        for i, l in enumerate(lines):
            if re.fullmatch(r"\d+:", l):
                labels.setdefault(l[:-1], []).append(i)

        def target(i, ref):
            n, d = ref[:-1], ref[-1]
            cands = labels[n]
            return min(j for j in cands if j > i) if d == "f" else max(j for j in cands if j < i)

        i, steps = 0, 0
        short = self.polls  # looks at a slot's counter that still find it short
        last_cmp = ""
        q = self.q
        while i < len(lines):
            steps += 1
            assert steps < 400000
            l = lines[i]
            op = l.split()[0] if l else ""
            args = [a.strip() for a in l[len(op):].split(",")] if l else []
            nxt = i + 1
            if op.startswith("s_cmp"):
                last_cmp = l
            if op == "s_waitcnt":
                self.wait(int(re.search(r"lgkmcnt\((\d+)\)", l).group(1)))
            elif op in ("ds_read_b128", "ds_read_b64_tr_b16"):
                dst, addr = args[0], args[1].split()[0]
                off = int(re.search(r"offset:(\d+)", l).group(1))
                tag = q[addr[2:-1]]
                if tag is None:
                    self.fail("read through an address register never set: " + l)
                elif tag >= self.iters:
                    self.fail("read of K-iteration %d, past the tile's %d" % (tag, self.iters))
                self.pending.append((regs(dst), tag, l))
                self.check_bounds(op, dst, addr, off)
            elif op == "ds_read_b32":
                self.pending.append((regs(args[0]), None, l))
            elif op == "ds_add_u32":
                u = q["rel"]  # releases the slot of K-iteration rel
                for w, tag, d in self.pending:
                    if tag == u:
                        self.fail("K-iteration %d's slot released while its read %s is outstanding" % (u, d))
                self.released.append(u)
                self.pending.append((set(), None, l))
            elif op.startswith("v_mfma"):
                self.need(regs(args[1]) | regs(args[2]), l)
            elif op == "v_readfirstlane_b32":
                self.need(regs(args[1]), l)
            elif op == "v_add_u32" and args[0] in ("%[va]", "%[vb]"):
                q[args[0][2:-1]] = q[args[1][2:-1]]
                if args[0] == "%[va]":
                    self.kss_a = 0
            elif op == "v_xor_b32" and args[0] == "%[va]":
                self.kss_a = int(args[1]) // 32
            elif op == "s_mul_i32" and args[0] == "%[rb]":
                assert args[1] == "%[rs]" and int(args[2]) == self.c.stage
                q["rb"] = q["rs"]
            elif op == "s_mov_b32" and args[1] == "%[slot]" and args[0] in ("%[rs]", "%[rel]"):
                q[args[0][2:-1]] = 0
            elif op == "s_add_u32" and args[0] == args[1] and args[0] in ("%[rs]", "%[rel]") and args[2] == "1":
                q[args[0][2:-1]] += 1
            elif op == "s_mov_b32" and args[0] == "%[slot]" and args[1] == "%[rs]":
                q["slot"] = q["rs"]
            elif op == "s_lshr_b32" and args[0] == "%[kk]":
                self.kk = self.iters >> int(args[2])
            elif op == "s_sub_u32" and args[0] == "%[kk]":
                self.kk -= 1
            elif op in ("s_cbranch_scc0", "s_cbranch_scc1", "s_branch"):
                ref = args[0]
                if op == "s_branch":
                    take = True
                elif "s_cmp_eq_u32 %[kk], 0" in last_cmp:       # straight to the last four k-steps
                    take = self.kk == 0
                elif "s_cmp_lg_u32 %[kk], 0" in last_cmp:       # loop back
                    take = self.kk != 0
                elif "%[dly]" in last_cmp:                      # no delay requested
                    take = True
                elif "s_cmp_ge_i32 %[t0], 0" in last_cmp:       # slot full?
                    take = short == 0
                    short = self.polls if take else short - 1
                elif "s_cmp_lg_u32 %[t0], 0" in last_cmp:       # abort flag up?
                    take = False
                elif "%[spins]" in last_cmp:                    # poll limit reached?
                    take = False
                else:
                    raise AssertionError("unknown branch condition: %s after %s" % (l, last_cmp))
                if take:
                    nxt = target(i, ref)
            i = nxt
        if any(w for w, _, _ in self.pending):
            self.fail("block ends with reads outstanding: %s" % [d for w, _, d in self.pending if w])

    def check_bounds(self, op, dst, addr, off):
        c = self.c
        r = sorted(regs(dst))
        if r[0] < c.frag_base or r[-1] > 255:
            self.fail("read into %s outside the fragment registers" % dst)
        if op == "ds_read_b128":
            assert addr == "%[va]"
            # row block mb of the A tile (rows 32 mb .. of the wave's tile)
            if off % (32 * c.tk * 2) or off // (32 * c.tk * 2) >= c.bm:
                self.fail("A read offset %d outside the wave's rows" % off)
        else:
            assert addr == "%[vb]"
            kq = off // 128 // c.nq  # B block row: k-rows 4 kq .. 4 kq + 3 of the tile
            if not 0 <= kq < c.tk // 4 or off >= c.tk * c.tn * 2:
                self.fail("B read offset %d outside the B tile" % off)
            elif kq // 4 != self.kss_a:
                self.fail("B read of k-step %d after A address of k-step %s" % (kq // 4, self.kss_a))


# polls: how many looks at each slot's counter find it short (0: the peeked
# value suffices; 1: the first poll succeeds; 2: a poll fails, the abort flag
# is read, and the next poll succeeds).  K-iterations per tile: every count
# the loop admits (S KS a multiple of 4) from no loop body up to five.
def iter_counts(key):
    ks = key[2] // 16
    return [n * 4 // ks for n in (1, 2, 3, 4, 6)]


CASES = [(k, iters, polls) for k in sorted(blocks()) for iters in iter_counts(k) for polls in (0, 1, 2)]


@pytest.mark.parametrize("key,iters,polls", CASES, ids=lambda v: str(v))
def test_every_wait_covers_what_follows(key, iters, polls):
    cfg = gen.Cfg(*key[:5])
    sim = Sim(cfg, iters, polls)
    sim.run(blocks()[key])
    assert not sim.errors, sim.errors[:5]
    assert sim.released == list(range(iters)), sim.released  # every K-iteration released once, in order
    assert sim.q["slot"] == iters  # hands the next tile's first K-iteration back


def test_committed_file_is_what_the_generator_writes():
    assert gen.main(["--check"]) == 0


def test_generator_covers_the_dispatched_configurations():
    keys = set(blocks())
    for t in gen.CONFIGS:
        assert t + (True,) in keys and t + (False,) in keys


@pytest.mark.parametrize("key", sorted(blocks()), ids=lambda v: str(v))
def test_checker_catches_a_weakened_wait(key):
    """The checker has teeth: waits below 15 made one weaker are caught on
    some path.  (The generator counts the operations younger than the one a
    wait needs without crediting earlier waits, so a wait that an earlier
    one already covers may pass weakened; at least three must be caught.)"""
    lines = blocks()[key]
    cfg = gen.Cfg(*key[:5])
    caught = 0
    for i, l in enumerate(lines):
        if not l.startswith("s_waitcnt"):
            continue
        n = int(re.search(r"\((\d+)\)", l).group(1))
        if n >= 15:
            continue  # all but the 15 youngest: the counter's limit
        bad = list(lines)
        bad[i] = "s_waitcnt lgkmcnt(%d)" % (n + 1)
        found = False
        for iters in iter_counts(key)[:3]:
            for polls in (0, 1, 2):
                sim = Sim(cfg, iters, polls)
                sim.run(bad)
                found |= bool(sim.errors)
        caught += found
    assert caught >= 3, caught
