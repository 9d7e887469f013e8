"""Static check of the generated K loop for two consumer waves per SIMD
(RollLoop in paper_2506_11209_amd/csrc/ws_deep_loop.inc: eight consumer waves
in a 2 x 4 grid, or four in a 2 x 2 grid at 128 x 128 x 32), CPU only.

The asm text of every configuration is executed by a small interpreter: the
scalar and address arithmetic run on concrete values for several lanes of
several consumer waves, LDS operations complete only when an s_waitcnt forces
them (in order), and the ring protocol is tracked (which K-iteration each slot
holds once its full counter has been checked, and which slot each release
frees).  Along every path a tile can take (1 to 5 K-iterations; each slot's
counter found full at the first look, after one poll, or after a failed
poll):

  * every read lands on the lane's own element of the operand layout: the A
    rows and k-chunk (through the XOR swizzle) or the B block and byte the
    MFMA fragment needs, inside the slot of a K-iteration already checked full;
  * every MFMA reads fragment registers that hold exactly the data of its own
    k-step, row block and column block, after their loads completed, and each
    accumulator takes its k-steps in order, once each;
  * a slot is released only after every read of its K-iteration completed,
    each K-iteration exactly once, in order;
  * nothing is in flight when the block ends, and the block hands back the
    slot and full-counter target of the next tile's first K-iteration.

A wait made one weaker is caught on some path."""
import os
import re
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2506_11209_amd", "csrc")
sys.path.insert(0, CSRC)
import gen_deep_loop as gen  # noqa: E402

HEADER = 256


def blocks():
    """{(tm, tn, tk, nc, np, bf16, traced): [asm lines]} of the RollLoop blocks
    (tile and its event-traced twin tile_traced)."""
    with open(gen.OUT) as f:
        text = f.read()
    out = {}
    for m in re.finditer(r"struct RollLoop<(\d+), (\d+), (\d+), (\d+), (\d+), (true|false)> \{(.*?)\n\};", text,
                         re.S):
        key = tuple(int(x) for x in m.groups()[:5]) + (m.group(6) == "true",)
        for fn in re.finditer(r"uint32_t (tile|tile_traced)\((.*?)return st;", m.group(7), re.S):
            lines = re.findall(r'^\s*"(.*)\\n\\t"$', fn.group(2), re.M)
            out[key + (fn.group(1) == "tile_traced",)] = [l.strip() for l in lines]
    return out


def swz_a(tk, r):
    """The kernels' XOR swizzle of A-tile row r (ws_gemm_kernel.hpp, swz_a)."""
    if tk == 32:
        return (r ^ (r >> 2)) & 3
    if tk == 64:
        return (r ^ ((r >> 3) & 1)) & 7
    return r & 15


def vregs(tok):
    m = re.fullmatch(r"v\[(\d+):(\d+)\]", tok)
    assert m, tok
    return list(range(int(m.group(1)), int(m.group(2)) + 1))


class Lane:
    """Lane `lane` of consumer wave `cw`: its operand offsets (as the C++
    caller computes them) and the operand elements it must read."""

    def __init__(self, c, cw, lane):
        self.c, self.cw, self.lane = c, cw, lane
        grid_n = 4 if c.nc == 8 else 2  # the kernel's consumer grid: two rows of NC / 2 waves
        self.wm, self.wn = cw // grid_n, cw % grid_n
        r = self.wm * c.wm + (lane & 31)
        self.a_off0 = r * c.tk * 2 + (((lane >> 5) ^ swz_a(c.tk, r)) << 4)
        g = lane >> 4
        self.b_off = (c.a_bytes + ((2 * (g >> 1)) * c.nq + (self.wn * c.wn) // 16 + (g & 1)) * 128 +
                      8 * (lane & 15))

    def decode_a(self, within):
        """(kss, mb) of an A read at byte `within` of a slot, or a message."""
        c = self.c
        if not 0 <= within < c.a_bytes:
            return "A read outside the A tile (byte %d)" % within
        row, pos = within // (c.tk * 2), (within % (c.tk * 2)) // 16
        if within % 16:
            return "A read not 16-byte aligned"
        chunk = pos ^ swz_a(c.tk, row)
        rr = row - self.wm * c.wm - (self.lane & 31)
        if rr % 32 or not 0 <= rr // 32 < c.bm:
            return "A read of row %d, not one of lane %d's rows" % (row, self.lane)
        k0 = 8 * chunk - 8 * (self.lane >> 5)
        if k0 % 16:
            return "A read of k-chunk %d, not lane %d's half of a k-step" % (chunk, self.lane)
        return (k0 // 16, rr // 32)

    def decode_b(self, within):
        """(kss, nb, half) of a transposed B read at byte `within` of a slot."""
        c = self.c
        boff = within - c.a_bytes
        if not 0 <= boff < c.tk * c.tn * 2:
            return "B read outside the B tile (byte %d)" % within
        block, byte = boff // 128, boff % 128
        if byte != 8 * (self.lane & 15):
            return "B read at byte %d of a block, not lane %d's" % (byte, self.lane)
        kq, nq = block // c.nq, block % c.nq
        g = self.lane >> 4
        rem = kq % 4 - 2 * (g >> 1)
        nrel = nq - (self.wn * c.wn) // 16 - (g & 1)
        if rem not in (0, 1) or nrel % 2 or not 0 <= nrel // 2 < c.bn:
            return "B read of block (%d, %d), not lane %d's" % (kq, nq, self.lane)
        return (kq // 4, nrel // 2, rem)


class Sim:
    def __init__(self, c, S, polls, lanes, P, slot0):
        self.c, self.S, self.polls, self.lanes, self.P = c, S, polls, lanes, P
        self.errors = []
        ring = HEADER
        self.s = {"slot": slot0, "ft": 4 * (1 + 0), "P": P, "S": S, "ring": ring, "fullb": 0,
                  "emptyb": 32, "abortb": 64, "lim": 1000, "dly": 0, "tq": 7, "tlim": 1000}
        self.vx = None
        self.stores = []          # (record index, event) of the trace stores, in order
        base = ring + slot0 * c.stage
        self.va = [base + ln.a_off0 for ln in lanes]
        self.vb = [base + ln.b_off for ln in lanes]
        self.pending = []        # [(regs, data tag or None, K-iteration or None, text)] oldest first
        self.data = {}           # fragment register -> data tag
        self.avail = [(0, slot0)]  # (K-iteration, slot) checked full and not yet released
        self.checked = 1
        self.released = []
        self.mfmas = 0
        self.acc_steps = {}

    def fail(self, msg):
        if len(self.errors) < 20:
            self.errors.append(msg)

    def wait(self, n):
        keep = self.pending[len(self.pending) - n:] if n else []
        for regs, tag, _, _ in self.pending[:len(self.pending) - len(keep)]:
            for r in regs:
                self.data[r] = tag
        self.pending = keep

    def val(self, tok):
        tok = tok.strip()
        m = re.fullmatch(r"%\[(\w+)\]", tok)
        if m:
            return self.s[m.group(1)]
        return int(tok, 0)

    def iter_of_slot(self, slot):
        its = [q for q, s in self.avail if s == slot]
        if len(its) != 1:
            return None
        return its[0]

    def read(self, op, dst, addr_reg, off, text):
        c = self.c
        regs = vregs(dst)
        tags = set()
        its = set()
        for i, ln in enumerate(self.lanes):
            addr = (self.va[i] if addr_reg == "va" else self.vb[i]) + off
            rel = addr - HEADER
            slot, within = rel // c.stage, rel % c.stage
            if not 0 <= slot < self.P:
                self.fail("%s: address outside the ring" % text)
                return
            q = self.iter_of_slot(slot)
            if q is None:
                self.fail("%s: slot %d holds no K-iteration checked full" % (text, slot))
                return
            its.add(q)
            if op == "ds_read_b128":
                d = ln.decode_a(within)
                if isinstance(d, str):
                    self.fail("%s (lane %d of wave %d): %s" % (text, ln.lane, ln.cw, d))
                    return
                tags.add((q, d[0], "A", d[1]))
            else:
                d = ln.decode_b(within)
                if isinstance(d, str):
                    self.fail("%s (lane %d of wave %d): %s" % (text, ln.lane, ln.cw, d))
                    return
                tags.add((q, d[0], "B", d[1], d[2]))
        if len(tags) != 1:
            self.fail("%s: lanes disagree on what they read: %s" % (text, tags))
            return
        tag = tags.pop()
        if op == "ds_read_b128":
            ok = regs == [c.frag_base + 4 * tag[3] + i for i in range(4)]
        else:
            b = c.frag_base + 4 * c.bm + 4 * tag[3] + 2 * tag[4]
            ok = regs == [b, b + 1]
        if not ok:
            self.fail("%s: data %s into the wrong registers" % (text, tag))
        self.pending.append((regs, tag, its.pop(), text))

    def mfma(self, args, text):
        c = self.c
        m = re.fullmatch(r"%\[c(\d+)_(\d+)\]", args[0])
        mb, nb = int(m.group(1)), int(m.group(2))
        t = self.mfmas // (c.bm * c.bn)
        q, kss = t // c.ks, t % c.ks
        self.mfmas += 1
        for regs, _, _, d in self.pending:
            if set(regs) & (set(vregs(args[1])) | set(vregs(args[2]))):
                self.fail("%s reads registers whose load %s is outstanding" % (text, d))
        want_a = (q, kss, "A", mb)
        for r in vregs(args[1]):
            if self.data.get(r) != want_a:
                self.fail("%s: A register v%d holds %s, wants %s" % (text, r, self.data.get(r), want_a))
                break
        breg = vregs(args[2])
        for h in (0, 1):
            want_b = (q, kss, "B", nb, h)
            for r in breg[2 * h:2 * h + 2]:
                if self.data.get(r) != want_b:
                    self.fail("%s: B register v%d holds %s, wants %s" % (text, r, self.data.get(r), want_b))
                    break
        prev = self.acc_steps.get((mb, nb), -1)
        if prev != t - 1:
            self.fail("%s: accumulator (%d, %d) takes k-step %d after %d" % (text, mb, nb, t, prev))
        self.acc_steps[(mb, nb)] = t

    def run(self, lines):
        labels = {}
        for i, l in enumerate(lines):
            if re.fullmatch(r"\d+:", l):
                labels.setdefault(l[:-1], []).append(i)

        def target(i, ref):
            n, d = ref[:-1], ref[-1]
            cands = labels[n]
            return min(j for j in cands if j > i) if d == "f" else max(j for j in cands if j < i)

        s = self.s
        i, steps = 0, 0
        short = self.polls
        last_cmp, scc = "", False
        while i < len(lines):
            steps += 1
            assert steps < 200000
            l = lines[i]
            op = l.split()[0] if l else ""
            args = [a.strip() for a in l[len(op):].split(",")] if l else []
            nxt = i + 1
            if op == "s_waitcnt":
                self.wait(int(re.search(r"lgkmcnt\((\d+)\)", l).group(1)))
            elif op in ("ds_read_b128", "ds_read_b64_tr_b16"):
                addr = args[1].split()[0]
                off = int(re.search(r"offset:(\d+)", l).group(1))
                self.read(op, args[0], addr[2:-1], off, l)
            elif op == "ds_read_b32":
                self.pending.append(([args[0]], None, None, l))
            elif op == "ds_add_u32":
                if not self.avail:
                    self.fail("release with no K-iteration held")
                else:
                    q, slot = self.avail[0]
                    if slot != s["rel"]:
                        self.fail("release of slot %d, but K-iteration %d holds slot %d" % (s["rel"], q, slot))
                    for _, _, qq, d in self.pending:
                        if qq == q:
                            self.fail("K-iteration %d released while its read %s is outstanding" % (q, d))
                    self.avail.pop(0)
                    self.released.append(q)
                self.pending.append(([], None, None, l))
            elif op.startswith("v_mfma"):
                self.mfma(args, l)
            elif op == "v_readfirstlane_b32":
                for regs, _, _, d in self.pending:
                    if args[1] in regs:
                        self.fail("%s before its load %s completed" % (l, d))
                s[args[0][2:-1]] = 0
            elif op == "v_add_u32" and args[0] in ("%[va]", "%[vb]"):
                d = self.val(args[1])
                arr = self.va if args[0] == "%[va]" else self.vb
                for k in range(len(arr)):
                    arr[k] = (arr[k] + d) & 0xFFFFFFFF
            elif op == "v_xor_b32" and args[0] == "%[va]":
                x = int(args[1])
                self.va = [v ^ x for v in self.va]
            elif op == "v_mov_b32":
                if args[0] == "%[vx]" and args[1].startswith("%["):
                    self.vx = self.val(args[1])
            elif op == "s_memtime":
                pass  # waited for by the s_waitcnt lgkmcnt(0) that follows it (checked below)
            elif op == "global_store_dword":
                assert args[0] == "%[vx]" and args[2] == "%[tr]", l
                self.stores.append((self.vx // 32, (self.vx % 32) // 4))
            elif op == "s_mov_b32":
                s[args[0][2:-1]] = self.val(args[1])
            elif op == "s_mov_b64":
                pass
            elif op == "s_add_u32":
                s[args[0][2:-1]] = (self.val(args[1]) + self.val(args[2])) & 0xFFFFFFFF
            elif op == "s_sub_u32":
                s[args[0][2:-1]] = (self.val(args[1]) - self.val(args[2])) & 0xFFFFFFFF
            elif op == "s_mul_i32":
                s[args[0][2:-1]] = (self.val(args[1]) * self.val(args[2])) & 0xFFFFFFFF
            elif op == "s_lshl_b32":
                s[args[0][2:-1]] = (self.val(args[1]) << self.val(args[2])) & 0xFFFFFFFF
            elif op == "s_cselect_b32":
                s[args[0][2:-1]] = self.val(args[1]) if scc else self.val(args[2])
            elif op.startswith("s_cmp"):
                last_cmp = l
                a, b = self.val(args[0]), self.val(args[1])
                scc = {"s_cmp_eq_u32": a == b, "s_cmp_lg_u32": a != b, "s_cmp_ge_i32": a >= b,
                       "s_cmp_gt_i32": a > b, "s_cmp_le_i32": a <= b, "s_cmp_lt_u32": a < b}[op]
            elif op in ("s_cbranch_scc0", "s_cbranch_scc1", "s_branch"):
                ref = args[0]
                if op == "s_branch":
                    take = True
                elif "s_cmp_ge_i32 %[t0], 0" in last_cmp:  # slot full?
                    take = short == 0
                    if take:
                        short = self.polls
                        self.avail.append((self.checked, s["rs"]))
                        self.checked += 1
                    else:
                        short -= 1
                elif "s_cmp_lg_u32 %[t0], 0" in last_cmp:  # abort flag up?
                    take = False
                elif "%[spins]" in last_cmp:  # poll limit reached?
                    take = False
                else:
                    take = scc if op == "s_cbranch_scc1" else not scc
                if take:
                    nxt = target(i, ref)
            elif op in ("s_nop", "s_sleep") or re.fullmatch(r"\d+:", l):
                pass
            else:
                raise AssertionError("the checker does not know %r" % l)
            i = nxt
        if self.pending:
            self.fail("block ends with operations in flight: %s" % [d for _, _, _, d in self.pending])


def iter_counts():
    return [1, 2, 3, 4, 5]


def lanes_of(c):
    waves = (0, 3, 5) if c.nc == 8 else (0, 1, 3)  # both grid rows, several columns
    return [Lane(c, cw, ln) for cw in waves for ln in (0, 1, 15, 16, 31, 32, 47, 63)]


CASES = [(k, S, polls, P) for k in sorted(blocks()) for S in iter_counts() for polls in (0, 1, 2)
         for P in ((2,) if k[2] == 64 else (2, 4))]


@pytest.mark.parametrize("key,S,polls,P", CASES, ids=lambda v: str(v))
def test_roll_block_reads_waits_and_releases(key, S, polls, P):
    c = gen.RollCfg(*key[:5])
    slot0 = 1 % P
    sim = Sim(c, S, polls, lanes_of(c), P, slot0)
    lines = blocks()[key]
    sim.run(lines)
    assert not sim.errors, sim.errors[:5]
    assert sim.mfmas == c.bm * c.bn * c.ks * S
    assert sim.released == list(range(S)), sim.released
    assert sim.s["st"] == 0
    assert sim.s["slot"] == (slot0 + S) % P
    assert sim.s["ft"] == 4 * (1 + (slot0 + S) // P)  # np = 4 signals per use of a slot
    if key[6]:
        # traced twin: per K-iteration u of the tile, record tq + u gets the
        # slot-full stamp (event 4, from the second K-iteration on: the caller
        # stores the first), then MFMAs under way (5), then released (6)
        tq = sim.s["tq"]
        want = []
        for u in range(S):
            want.append((tq + u, 5))
            if u + 1 < S:
                want.append((tq + u + 1, 4))
            want.append((tq + u, 6))
        assert sim.stores == want, sim.stores
        for i, l in enumerate(lines):  # every timer read is waited for at once
            if l.startswith("s_memtime"):
                assert lines[i + 1] == "s_waitcnt lgkmcnt(0)"
    else:
        assert not sim.stores and not any(l.startswith("s_memtime") for l in lines)


def test_generator_covers_the_dispatched_configurations():
    keys = set(blocks())
    for t in gen.ROLL_CONFIGS:
        for bf16 in (True, False):
            for traced in (False, True):
                assert t + (bf16, traced) in keys


@pytest.mark.parametrize("key", sorted(blocks()), ids=lambda v: str(v))
def test_checker_catches_a_weakened_wait(key):
    lines = blocks()[key]
    c = gen.RollCfg(*key[:5])
    caught = total = 0
    for i, l in enumerate(lines):
        if not l.startswith("s_waitcnt"):
            continue
        n = int(re.search(r"\((\d+)\)", l).group(1))
        if n >= 15 or i + 1 == len(lines) or "s_nop" in lines[i + 1]:
            continue
        if lines[i - 1].startswith("s_memtime"):
            continue  # the timer's own wait (checked in the main test)
        j = i - 1
        while j >= 0 and not lines[j].startswith(("ds_", "s_waitcnt")):
            j -= 1
        if j >= 0 and lines[j] == "s_waitcnt lgkmcnt(0)":
            continue  # nothing issued since a full drain: the wait is already met
        total += 1
        bad = list(lines)
        bad[i] = "s_waitcnt lgkmcnt(%d)" % (n + 1)
        found = False
        for S in (1, 2, 3):
            for polls in (0, 2):
                sim = Sim(c, S, polls, lanes_of(c)[:2], 2, 1)
                sim.run(bad)
                found |= bool(sim.errors)
        caught += found
    assert total >= 10 and caught >= total - 2, (caught, total)
