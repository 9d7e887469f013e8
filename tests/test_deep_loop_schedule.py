"""Static check of the hand-placed LDS waits in the generated deep-prefetch K
loop (paper_2506_11209_amd/csrc/ws_deep_loop.inc).

The asm text of every configuration is interpreted along each path a tile
can take (1, 2, 3 and 6 K-iterations; the next slot's counter found full at
the first look, or only after polling) under the most pessimistic timing a
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
    a wait forces them."""

    def __init__(self, cfg, iters, polls):
        self.c, self.iters, self.polls = cfg, iters, polls
        self.released = []
        self.pending = []  # [(registers written, slot tag, description)] oldest first
        self.q = {"slot": 0, "ns": 1, "base": 0, "nbase": None, "va": None, "vb": None}
        self.kk = None
        self.errors = []

    def fail(self, msg):
        self.errors.append(msg)

    def wait(self, n):
        keep = self.pending[len(self.pending) - n:] if n else []
        self.pending = keep

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
        short = self.polls  # looks at the next slot's counter that still find it short
        last_cmp = ""
        while i < len(lines):
            steps += 1
            assert steps < 200000
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
                tag = self.q[addr[2:-1]]
                if tag is None:
                    self.fail("read through an address register never set: " + l)
                self.pending.append((regs(dst), tag, l))
                self.check_bounds(op, dst, addr, off)
            elif op == "ds_read_b32":
                self.pending.append((regs(args[0]), None, l))
            elif op == "ds_add_u32":
                slot = self.q["slot"]  # releases the slot in %[slot]
                for w, tag, d in self.pending:
                    if tag == slot:
                        self.fail("slot %d released while its read %s is outstanding" % (slot, d))
                self.released.append(slot)
            elif op.startswith("v_mfma"):
                self.need(regs(args[1]) | regs(args[2]), l)
            elif op == "v_readfirstlane_b32":
                self.need(regs(args[1]), l)
            elif op == "v_add_u32" and args[0] in ("%[va]", "%[vb]"):
                self.q[args[0][2:-1]] = self.q[args[1][2:-1]]
            elif op == "s_mul_i32" and args[0] == "%[nbase]":
                self.q["nbase"] = self.q["ns"]
            elif op == "s_mov_b32" and args[0] == "%[base]" and args[1] == "%[nbase]":
                self.q["base"] = self.q["nbase"]
            elif op == "s_mov_b32" and args[0] == "%[slot]" and args[1] == "%[ns]":
                self.q["slot"] = self.q["ns"]
                self.q["ns"] = self.q["slot"] + 1
            elif op == "s_sub_u32" and args[0] == "%[kk]":
                self.kk = self.iters - 1 if args[1] == "%[S]" else self.kk - 1
            elif op in ("s_cbranch_scc0", "s_cbranch_scc1", "s_branch"):
                ref = args[0]
                if op == "s_branch":
                    take = True
                elif "%[S], 1" in last_cmp:                    # skip the peek when S == 1
                    take = not (self.iters > 1)
                elif "s_cmp_eq_u32 %[kk], 0" in last_cmp:       # straight to the last K-iteration
                    take = self.kk == 0
                elif "s_cmp_lg_u32 %[kk], 0" in last_cmp:       # loop back
                    take = self.kk != 0
                elif "%[dly]" in last_cmp:                      # no delay requested
                    take = True
                elif "s_cmp_ge_i32 %[t0], 0" in last_cmp:       # next slot full?
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
        if self.pending:
            self.fail("block ends with reads outstanding: %s" % [d for _, _, d in self.pending])

    def check_bounds(self, op, dst, addr, off):
        c = self.c
        r = sorted(regs(dst))
        if r[0] < c.frag_base or r[-1] > 255:
            self.fail("read into %s outside the fragment registers" % dst)
        s = (r[0] - c.frag_base) // c.set_regs
        if op == "ds_read_b128":
            assert addr == "%[va]"
            # row block mb of the A tile (rows 32 mb .. of the wave's tile)
            if off % (32 * c.tk * 2) or off // (32 * c.tk * 2) >= c.bm:
                self.fail("A read offset %d outside the wave's rows" % off)
        else:
            assert addr == "%[vb]"
            kq = off // 128 // c.nq
            if not (4 * s <= kq < 4 * s + 4):
                self.fail("B read offset %d outside k-step %d" % (off, s))
            if off >= c.tk * c.tn * 2:
                self.fail("B read offset %d past the B tile" % off)


# polls: how many looks at each next slot's counter find it short (0: the
# peeked value suffices; 1: the first poll succeeds; 2: a poll fails, the
# abort flag is read, and the next poll succeeds)
CASES = [(k, iters, polls) for k in sorted(blocks()) for iters in (1, 2, 3, 6) for polls in (0, 1, 2)]


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
    """The checker has teeth: the waits that are exact (no younger operation
    to spare on some path), made one weaker, are caught.  Waits with slack
    (the steady K-iteration's first wait has two more younger operations
    than it needs) may pass weakened."""
    lines = blocks()[key]
    cfg = gen.Cfg(*key[:5])
    exact = {cfg.reads, 0}  # last K-iteration: R younger at k-step 2, none at k-step 3
    caught, exact_seen = 0, 0
    for i, l in enumerate(lines):
        if not l.startswith("s_waitcnt"):
            continue
        n = int(re.search(r"\((\d+)\)", l).group(1))
        if n >= 15:
            continue  # all but the 15 youngest: the counter's limit
        bad = list(lines)
        bad[i] = "s_waitcnt lgkmcnt(%d)" % (n + 1)
        found = False
        for iters in (1, 2, 3):
            for polls in (0, 1, 2):
                sim = Sim(cfg, iters, polls)
                sim.run(bad)
                found |= bool(sim.errors)
        caught += found
        if n in exact:
            exact_seen += 1
            assert found, "weakening the exact wait %s was not caught" % l
    assert exact_seen >= 3 and caught >= exact_seen
