"""Generate ws_deep_loop.inc: the K loop of one output tile for the
deep-prefetch consumer, as one asm block per kernel configuration.

    python paper_2506_11209_amd/csrc/gen_deep_loop.py            # rewrite the .inc
    python paper_2506_11209_amd/csrc/gen_deep_loop.py --check    # exit 1 if it is stale

Why asm: the consumer keeps three k-steps of LDS operand reads in flight
behind its MFMAs.  Written in C++ the compiler either waits for every read
at the loop head (its wait analysis) or, with the reads hidden in asm,
copies and spills the fragment registers while their reads are still in
flight.  Here the fragments live in fixed registers at the top of the
register file (clobbered by the block), the accumulators are operands, and
every LDS wait is placed by hand.

The schedule, per k-step t of a tile (T = S KS k-steps, KS = TK / 16 per
K-iteration, one 32x32x16 MFMA per 32x32 block and k-step):

  * wait until the reads of k-step t have landed;
  * if k-step t + 3 exists: when it starts a new K-iteration, check that
    K-iteration's slot is full (its counter was peeked when the read stream
    entered the previous slot; poll, draining every read, only when it is
    short) and peek at the slot after it; then issue the reads of k-step
    t + 3, one ahead of each MFMA of k-step t;
  * when t + 2 ends a K-iteration (t = (u + 1) KS - 2 for K-iteration u),
    release u's slot: its last reads, for k-step (u + 1) KS - 1, went out at
    k-step t - 2.

Fragment set s = t mod 4 holds BM A fragments (ds_read_b128) and BN B
fragments (two ds_read_b64_tr_b16 each).  The loop body is four k-steps
(4 / KS K-iterations, so a tile needs S KS divisible by 4), preceded by a
prologue (the reads of k-steps 0-2) and followed by the tile's last four
k-steps, which read nothing ahead.  A wave's LDS operations complete in
order, so every wait is "at most n younger LDS operations outstanding"; the
generator derives each n by replaying the emitted operations along every
path through the block (prologue, then no loop body up to three, then the
last four k-steps) and keeping the tightest, capped at 15, the counter's
range.  The tests replay the emitted text independently.
"""
from __future__ import annotations

import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
OUT = os.path.join(HERE, "ws_deep_loop.inc")

# (TM, TN, TK, NC, SPLIT): the configurations that get the deep consumer
# (four consumer waves in a 2 x 2 grid).  Its fixed fragment registers make a
# kernel take all of a wave's registers (256 with one producer group, 168
# with two).  Left out because they measured slower with it (8192^3):
# 128x128x32 1:1 (6 %: one workgroup per CU where the compiler-scheduled
# kernel runs two; it takes the register-lean roll loop below, which keeps
# two), 64x128x32 and 128x64x32 1:1 (7-8 %); the 2:1 kernels of the largest
# tiles run the register-lean consumer.
# (TM, TN, TK, NC, NP): NP producer waves.  Four producer waves serve both
# the 1:1 arrangement and the 2:1 one with two groups of two (the consumer
# side is the same); eight are the 2:1 arrangement with two groups of four.
CONFIGS = [
    (256, 128, 64, 4, 4), (128, 256, 64, 4, 4), (128, 128, 64, 4, 4), (64, 128, 64, 4, 4),
    (128, 64, 64, 4, 4), (128, 256, 32, 4, 4),
    (128, 128, 64, 4, 8), (128, 64, 64, 4, 8), (64, 128, 64, 4, 8), (64, 64, 64, 4, 8),
    (128, 128, 32, 4, 8), (128, 64, 32, 4, 8), (64, 128, 32, 4, 8), (64, 64, 32, 4, 8),
]
HEADER_BYTES = 256
LGKM_MAX = 15


class Cfg:
    def __init__(self, tm, tn, tk, nc, np):
        assert nc == 4 and np in (4, 8) and tk in (32, 64)
        self.tm, self.tn, self.tk, self.nc, self.np = tm, tn, tk, nc, np
        self.ks = tk // 16                            # k-steps per K-iteration
        self.wm, self.wn = tm // 2, tn // 2
        self.bm, self.bn = self.wm // 32, self.wn // 32
        self.nq = tn // 16
        self.a_bytes = tm * tk * 2
        self.stage = self.a_bytes + tk * tn * 2
        self.reads = self.bm + 2 * self.bn            # LDS instructions per fragment set
        self.set_regs = 4 * (self.bm + self.bn)
        # a wave's registers: 256 with two waves per SIMD (4 + 4), 168 with three (4 + 8)
        self.vgprs = 256 if nc + self.np <= 8 else 168
        self.frag_base = self.vgprs - 4 * self.set_regs  # four sets at the top of the file
        assert self.reads <= LGKM_MAX and self.bm * self.bn * 16 + 4 * self.set_regs <= self.vgprs - 32
        assert self.stage % 128 == 0 and HEADER_BYTES % 128 == 0 and 4 % self.ks == 0


class Emitter:
    """Collects the asm lines of one pass over the block and the tags of its
    LDS operations in issue order.  A dry run records, for every wait site,
    how many operations are younger than the last one the site needs; the
    final pass writes the tightest count over all dry runs."""

    def __init__(self, waits=None):
        self.lines = []
        self.ops = []               # tags of LDS operations, oldest first
        self.waits = waits          # site -> lgkmcnt (final pass) or None (dry run)
        self.need = {}              # site -> tightest count seen (dry run)

    def emit(self, line):
        self.lines.append(line)

    def op(self, line, tag):
        self.lines.append(line)
        self.ops.append(tag)

    def wait_for(self, site, pred):
        """s_waitcnt so that every issued operation whose tag satisfies pred
        has completed."""
        if self.waits is None:
            idx = [i for i, t in enumerate(self.ops) if pred(t)]
            younger = len(self.ops) - 1 - idx[-1] if idx else LGKM_MAX
            self.need[site] = min(self.need.get(site, LGKM_MAX), younger)
            self.emit("s_waitcnt lgkmcnt(?)")
        else:
            self.emit("s_waitcnt lgkmcnt(%d)" % self.waits[site])


def program(E: Emitter, c: Cfg, bf16: bool, S: int | None):
    """Emit the block.  With S given (a dry run) the loop body is repeated as
    a tile of S K-iterations runs it, with absolute k-step numbers in the
    tags; with S None every segment is emitted once."""
    mfma = "v_mfma_f32_32x32x16_bf16" if bf16 else "v_mfma_f32_32x32x16_f16"
    KS = c.ks
    emit = E.emit

    def a_reg(s, mb):
        b = c.frag_base + s * c.set_regs + 4 * mb
        return "v[%d:%d]" % (b, b + 3)

    def b_regs(s, nb):
        b = c.frag_base + s * c.set_regs + 4 * c.bm + 4 * nb
        return "v[%d:%d]" % (b, b + 3), "v[%d:%d]" % (b, b + 1), "v[%d:%d]" % (b + 2, b + 3)

    def addr(kss):
        # address registers for k-step kss of the slot at SGPR rb: the A chunk
        # of k-step kss is (2 kss + lane / 32) ^ swz(row), i.e. bits 5.. of the
        # k-step 0 offset XORed by 32 kss (slots start on 128-byte boundaries)
        emit("v_add_u32 %[va], %[rb], %[aoff]")
        if kss:
            emit("v_xor_b32 %%[va], %d, %%[va]" % (32 * kss))
        emit("v_add_u32 %[vb], %[rb], %[boff]")

    def reads(t):
        # (line, tag) of the reads of k-step t into fragment set t mod 4
        s, kss = t % 4, t % KS
        out = []
        for mb in range(c.bm):
            off = mb * 32 * c.tk * 2
            assert off < 65536
            out.append(("ds_read_b128 %s, %%[va] offset:%d" % (a_reg(s, mb), off), ("R", t)))
        for nb in range(c.bn):
            _, lo, hi = b_regs(s, nb)
            off = ((4 * kss) * c.nq + 2 * nb) * 128
            assert off + c.nq * 128 < 65536
            out.append(("ds_read_b64_tr_b16 %s, %%[vb] offset:%d" % (lo, off), ("R", t)))
            out.append(("ds_read_b64_tr_b16 %s, %%[vb] offset:%d" % (hi, off + c.nq * 128), ("R", t)))
        return out

    def mfma_list(t):
        s = t % 4
        return ["%s %%[c%d_%d], %s, %s, %%[c%d_%d]" % (mfma, mb, nb, a_reg(s, mb), b_regs(s, nb)[0], mb, nb)
                for mb in range(c.bm) for nb in range(c.bn)]

    def next_slot(slot, target, tmp):
        # (slot, target) <- those of the next K-iteration: slot + 1 mod P, target + NP on wrap
        emit("s_add_u32 %%[%s], %%[%s], 1" % (slot, slot))
        emit("s_add_u32 %%[%s], %%[%s], %d" % (tmp, target, c.np))
        emit("s_cmp_eq_u32 %%[%s], %%[P]" % slot)
        emit("s_cselect_b32 %%[%s], 0, %%[%s]" % (slot, slot))
        emit("s_cselect_b32 %%[%s], %%[%s], %%[%s]" % (target, tmp, target))

    def peek(u):
        # issue a read of full[next(rs)], the counter of K-iteration u, into vp
        emit("s_add_u32 %[t1], %[rs], 1")
        emit("s_cmp_eq_u32 %[t1], %[P]")
        emit("s_cselect_b32 %[t1], 0, %[t1]")
        emit("s_lshl_b32 %[t1], %[t1], 2")
        emit("s_add_u32 %[t1], %[t1], %[fullb]")
        emit("v_mov_b32 %[vx], %[t1]")
        E.op("ds_read_b32 %[vp], %[vx]", ("peek", u))

    def check(site, u):
        # K-iteration u (slot rs, target rt) must be full; vp holds its peeked counter
        E.wait_for(site, lambda tag: tag == ("peek", u))
        emit("v_readfirstlane_b32 %[t0], %[vp]")
        emit("s_sub_u32 %[t0], %[t0], %[rt]")
        emit("s_cmp_ge_i32 %[t0], 0")
        emit("s_cbranch_scc1 2f")
        emit("s_mov_b32 %[spins], 0")
        emit("s_lshl_b32 %[t1], %[rs], 2")
        emit("s_add_u32 %[t1], %[t1], %[fullb]")
        emit("3:")
        emit("v_mov_b32 %[vx], %[t1]")
        emit("ds_read_b32 %[vp], %[vx]")
        emit("v_mov_b32 %[vx], %[abortb]")
        emit("ds_read_b32 %[vq], %[vx]")
        emit("s_waitcnt lgkmcnt(0)")
        emit("v_readfirstlane_b32 %[t0], %[vp]")
        emit("s_sub_u32 %[t0], %[t0], %[rt]")
        emit("s_cmp_ge_i32 %[t0], 0")
        emit("s_cbranch_scc1 2f")
        emit("v_readfirstlane_b32 %[t0], %[vq]")
        emit("s_cmp_lg_u32 %[t0], 0")
        emit("s_mov_b32 %[st], 1")
        emit("s_cbranch_scc1 9f")
        emit("s_add_u32 %[spins], %[spins], 1")
        emit("s_cmp_gt_i32 %[spins], %[lim]")
        emit("s_mov_b32 %[st], 2")
        emit("s_cbranch_scc1 9f")
        emit("s_sleep 1")
        emit("s_branch 3b")
        emit("2:")
        emit("s_mov_b32 %[st], 0")  # a poll may have set it before a branch not taken

    def enter(site, u):
        # the read stream moves on to K-iteration u > 0 of the tile
        next_slot("rs", "rt", "t0")
        check(site, u)
        emit("s_mul_i32 %%[rb], %%[rs], %d" % c.stage)
        emit("s_add_u32 %[rb], %[rb], %[ring]")
        peek(u + 1)

    def release(site, u):
        # K-iteration u's slot (SGPR rel) back to the producers once its reads landed
        E.wait_for(site, lambda tag: tag[0] == "R" and tag[1] // KS == u)
        emit("s_lshl_b32 %[t1], %[rel], 2")
        emit("s_add_u32 %[t1], %[t1], %[emptyb]")
        emit("v_mov_b32 %[vx], %[t1]")
        emit("v_mov_b32 %[vq], 1")
        emit("s_mov_b64 %[sav], exec")
        emit("s_mov_b64 exec, 1")
        E.op("ds_add_u32 %[vx], %[vq]", ("rel", u))
        emit("s_mov_b64 exec, %[sav]")
        emit("s_add_u32 %[rel], %[rel], 1")
        emit("s_cmp_eq_u32 %[rel], %[P]")
        emit("s_cselect_b32 %[rel], 0, %[rel]")

    def delay():
        emit("s_cmp_le_i32 %[dly], 0")
        emit("s_cbranch_scc1 6f")
        emit("s_mov_b32 %[t0], %[dly]")
        emit("5:")
        emit("s_sleep 127")
        emit("s_sub_u32 %[t0], %[t0], 1")
        emit("s_cmp_lg_u32 %[t0], 0")
        emit("s_cbranch_scc1 5b")
        emit("6:")

    def kstep(seg, t, read_ahead):
        # k-step t; read_ahead: k-step t + 3 exists
        E.wait_for((seg, t % 4, "R"), lambda tag: tag == ("R", t))
        ms = mfma_list(t)
        if read_ahead:
            if (t + 3) % KS == 0:
                enter((seg, t % 4, "enter"), (t + 3) // KS)
            addr((t + 3) % KS)
            rs = reads(t + 3)
            # read, MFMA, read, MFMA, ...: a wave tracks at most 15 LDS
            # operations, so a read can stall at issue; an MFMA after each keeps
            # the matrix core fed meanwhile (measured faster than issuing a
            # set's reads together, before or after its MFMAs)
            while ms or rs:
                if rs:
                    E.op(*rs.pop(0))
                if ms:
                    emit(ms.pop(0))
        else:
            for m in ms:
                emit(m)
        if (t + 2) % KS == 0:
            release((seg, t % 4, "rel"), (t + 2) // KS - 1)

    T = S * KS if S is not None else None
    # entry: the caller has waited for the tile's first slot (slot, ft); the
    # accumulators were just written by VALU instructions
    emit("s_nop 7")
    emit("s_mov_b32 %[st], 0")
    emit("s_mov_b32 %[rs], %[slot]")
    emit("s_mov_b32 %[rt], %[ft]")
    emit("s_mov_b32 %[rel], %[slot]")
    emit("s_mul_i32 %%[rb], %%[rs], %d" % c.stage)
    emit("s_add_u32 %[rb], %[rb], %[ring]")
    peek(1)
    # prologue: the reads of k-steps 0, 1 and 2
    for t in range(3):
        if t and t % KS == 0:
            enter(("pro", t, "enter"), t // KS)
        addr(t % KS)
        for line, tag in reads(t):
            E.op(line, tag)
    # S KS / 4 groups of four k-steps: the loop bodies, then the last group
    emit("s_lshr_b32 %%[kk], %%[S], %d" % {4: 0, 2: 1}[KS])
    emit("s_sub_u32 %[kk], %[kk], 1")
    emit("s_cmp_eq_u32 %[kk], 0")
    emit("s_cbranch_scc1 8f")
    emit("1:")
    for b in range((T // 4 - 1) if S is not None else 1):
        delay()
        for j in range(4):
            kstep("body", 4 * b + j, True)
    emit("s_sub_u32 %[kk], %[kk], 1")
    emit("s_cmp_lg_u32 %[kk], 0")
    emit("s_cbranch_scc1 1b")
    # the tile's last four k-steps: only the first reads ahead
    emit("8:")
    delay()
    t_last = (T - 4) if S is not None else 0
    for j in range(4):
        kstep("tail", t_last + j, j == 0)
    # hand back the slot and target of the next tile's first K-iteration
    next_slot("rs", "rt", "t0")
    emit("s_mov_b32 %[slot], %[rs]")
    emit("s_mov_b32 %[ft], %[rt]")
    emit("9:")
    # the caller reads the accumulators with VALU instructions
    for _ in range(3):
        emit("s_nop 15")


def tile_iters(c: Cfg):
    """K-iterations per tile replayed by the dry runs: no loop body, one, two
    and three (S KS must be a multiple of 4)."""
    return [n * 4 // c.ks for n in (1, 2, 3, 4)]


def gen_block(c: Cfg, bf16: bool) -> list[str]:
    waits = {}
    for S in tile_iters(c):
        E = Emitter()
        program(E, c, bf16, S)
        for site, n in E.need.items():
            waits[site] = min(waits.get(site, LGKM_MAX), n)
    E = Emitter(waits)
    program(E, c, bf16, None)
    return E.lines


def gen_struct(c: Cfg, bf16: bool) -> str:
    lines = gen_block(c, bf16)
    acc_ops = ", ".join('[c%d_%d] "+v"(c[%d][%d])' % (mb, nb, mb, nb) for mb in range(c.bm) for nb in range(c.bn))
    clobbers = ", ".join('"v%d"' % r for r in range(c.frag_base, c.vgprs))
    body = "\n".join('        "%s\\n\\t"' % l for l in lines)
    return """template <>
struct DeepLoop<%(tm)d, %(tn)d, %(tk)d, %(nc)d, %(np)d, %(bf16)s> {
  static constexpr bool kAvailable = true;
  static constexpr int kIterQuantum = %(quantum)d;  // K-iterations per tile: a multiple of this
  static __device__ __forceinline__ uint32_t tile(f32x16_t (&c)[%(bm)d][%(bn)d], uint32_t a_off0, uint32_t b_off,
                                                  uint32_t& slot, uint32_t& ftarget, uint32_t P, uint32_t S,
                                                  uint32_t ring, uint32_t fullb, uint32_t emptyb, uint32_t abortb,
                                                  int32_t lim, int32_t dly) {
#if defined(__HIP_DEVICE_COMPILE__)
    uint32_t st, rs, rt, rb, rel, kk, t0, t1, spins, va, vb, vp, vq, vx;
    uint64_t sav;
    asm volatile(
%(body)s
        : %(acc)s, [slot] "+s"(slot), [ft] "+s"(ftarget), [st] "=&s"(st), [rs] "=&s"(rs), [rt] "=&s"(rt),
          [rb] "=&s"(rb), [rel] "=&s"(rel), [kk] "=&s"(kk), [t0] "=&s"(t0), [t1] "=&s"(t1),
          [spins] "=&s"(spins), [sav] "=&s"(sav), [va] "=&v"(va), [vb] "=&v"(vb), [vp] "=&v"(vp),
          [vq] "=&v"(vq), [vx] "=&v"(vx)
        : [aoff] "v"(a_off0), [boff] "v"(b_off), [P] "s"(P), [S] "s"(S), [ring] "s"(ring),
          [fullb] "s"(fullb), [emptyb] "s"(emptyb), [abortb] "s"(abortb), [lim] "s"(lim), [dly] "s"(dly)
        : "memory", "scc", %(clobbers)s);
    return st;
#else
    (void)c; (void)a_off0; (void)b_off; (void)slot; (void)ftarget; (void)P; (void)S; (void)ring;
    (void)fullb; (void)emptyb; (void)abortb; (void)lim; (void)dly;
    return 0;
#endif
  }
};
""" % dict(tm=c.tm, tn=c.tn, tk=c.tk, nc=c.nc, np=c.np, bf16="true" if bf16 else "false", bm=c.bm,
           bn=c.bn, body=body, acc=acc_ops, clobbers=clobbers, quantum=4 // c.ks)


# ---------------------------------------------------------------------------
# Register-lean loop for two consumer waves per SIMD.  Eight consumer waves
# (2 x 4 grid) next to four producer waves: twelve waves leave 168 registers a
# wave, 128 of them the 128 x 64 accumulator.  Four consumer waves (2 x 2
# grid) next to four producer waves at 128 x 128 x 32: the kernel is held to
# 128 registers a wave so that two workgroups share a CU (sixteen waves), 64
# of them the 64 x 64 accumulator.  Either way each fragment is single-buffered
# and refilled right after its last MFMA of the k-step; the other consumer
# wave on the SIMD keeps the matrix core busy while one waits for a read.
#
# Per k-step t (N-major MFMA order, B fragment nb used by BM consecutive
# MFMAs, A fragment mb by MFMAs mb and BM + mb):
#   mfma(0..BM-1, 0); [enter the next slot if t + 1 starts a K-iteration]
#   read B(t + 1)[0]; mfma(0, 1); [release if t ends a K-iteration]
#   then mfma(mb, 1), read A(t + 1)[mb] for every mb; read B(t + 1)[1] ...
# so every read is at least BM - 1 MFMAs of this wave ahead of its use.
# The A address va and the B address vb move with the read stream: XOR of
# the k-step bits for A, the slot's byte delta for both.
# ---------------------------------------------------------------------------
# (TM, TN, TK, NC, NP)
ROLL_CONFIGS = [(256, 256, 64, 8, 4), (256, 256, 32, 8, 4), (128, 128, 32, 4, 4)]


class RollCfg:
    def __init__(self, tm, tn, tk, nc, np):
        assert nc in (4, 8) and np == 4 and tk in (32, 64)
        self.tm, self.tn, self.tk, self.nc, self.np = tm, tn, tk, nc, np
        self.ks = tk // 16
        self.wgn = 4 if nc == 8 else 2                # consumer grid columns (two rows)
        self.wm, self.wn = tm // 2, tn // self.wgn
        self.bm, self.bn = self.wm // 32, self.wn // 32
        self.nq = tn // 16
        self.a_bytes = tm * tk * 2
        self.stage = self.a_bytes + tk * tn * 2
        # registers a wave: 168 with twelve waves, 128 with two workgroups of eight
        self.vgprs = 168 if nc == 8 else 128
        self.frag_regs = 4 * (self.bm + self.bn)
        self.frag_base = self.vgprs - self.frag_regs
        assert self.bn == 2 and self.bm * self.bn * 16 + self.frag_regs <= self.vgprs - 8
        assert self.stage % 128 == 0 and HEADER_BYTES % 128 == 0


# XOR that moves an A address from k-step a to k-step b of a slot
def _kxor(a, b):
    return 32 * (a ^ b)


def program_roll(E: Emitter, c: RollCfg, bf16: bool, S: int | None, traced: bool = False):
    """Emit the roll block (see above).  With S given (a dry run) the loop body
    is repeated once per K-iteration with absolute k-step numbers in the tags.

    traced: the event-trace twin (consumer wave 0 of traced workgroups).  Per
    K-iteration u it stores three shader-clock stamps (s_memtime, low 32 bits)
    into the record of K-iteration tq + u of the trace buffer: the slot seen
    full (event 4, at the check of u), the MFMAs of u under way (event 5, after
    its first k-step's first MFMA column) and the slot released (event 6).
    Each stamp waits for every LDS operation of the wave (the timer is a
    scalar load and shares their counter); the stamps sit where at most two
    reads are outstanding, and those two are waited for right after anyway,
    except at the release."""
    mfma = "v_mfma_f32_32x32x16_bf16" if bf16 else "v_mfma_f32_32x32x16_f16"
    KS = c.ks
    emit = E.emit

    def a_reg(mb):
        b = c.frag_base + 4 * mb
        return "v[%d:%d]" % (b, b + 3)

    def b_reg(nb, part=None):
        b = c.frag_base + 4 * c.bm + 4 * nb
        if part is None:
            return "v[%d:%d]" % (b, b + 3)
        return "v[%d:%d]" % (b + 2 * part, b + 2 * part + 1)

    def read_a(t, mb):
        E.op("ds_read_b128 %s, %%[va] offset:%d" % (a_reg(mb), mb * 32 * c.tk * 2), ("A", t, mb))

    def read_b(t, nb):
        off = ((4 * (t % KS)) * c.nq + 2 * nb) * 128
        E.op("ds_read_b64_tr_b16 %s, %%[vb] offset:%d" % (b_reg(nb, 0), off), ("B", t, nb))
        E.op("ds_read_b64_tr_b16 %s, %%[vb] offset:%d" % (b_reg(nb, 1), off + c.nq * 128), ("B", t, nb))

    def mf(mb, nb):
        emit("%s %%[c%d_%d], %s, %s, %%[c%d_%d]" % (mfma, mb, nb, a_reg(mb), b_reg(nb), mb, nb))

    def next_slot(slot, target, tmp):
        emit("s_add_u32 %%[%s], %%[%s], 1" % (slot, slot))
        emit("s_add_u32 %%[%s], %%[%s], %d" % (tmp, target, c.np))
        emit("s_cmp_eq_u32 %%[%s], %%[P]" % slot)
        emit("s_cselect_b32 %%[%s], 0, %%[%s]" % (slot, slot))
        emit("s_cselect_b32 %%[%s], %%[%s], %%[%s]" % (target, tmp, target))

    def peek(u):
        emit("s_add_u32 %[t1], %[rs], 1")
        emit("s_cmp_eq_u32 %[t1], %[P]")
        emit("s_cselect_b32 %[t1], 0, %[t1]")
        emit("s_lshl_b32 %[t1], %[t1], 2")
        emit("s_add_u32 %[t1], %[t1], %[fullb]")
        emit("v_mov_b32 %[vx], %[t1]")
        E.op("ds_read_b32 %[vp], %[vx]", ("peek", u))

    def check(site, u):
        E.wait_for(site, lambda tag: tag == ("peek", u))
        emit("v_readfirstlane_b32 %[t0], %[vp]")
        emit("s_sub_u32 %[t0], %[t0], %[rt]")
        emit("s_cmp_ge_i32 %[t0], 0")
        emit("s_cbranch_scc1 2f")
        emit("s_mov_b32 %[spins], 0")
        emit("s_lshl_b32 %[t1], %[rs], 2")
        emit("s_add_u32 %[t1], %[t1], %[fullb]")
        emit("3:")
        emit("v_mov_b32 %[vx], %[t1]")
        emit("ds_read_b32 %[vp], %[vx]")
        emit("v_mov_b32 %[vx], %[abortb]")
        emit("ds_read_b32 %[vq], %[vx]")
        emit("s_waitcnt lgkmcnt(0)")
        emit("v_readfirstlane_b32 %[t0], %[vp]")
        emit("s_sub_u32 %[t0], %[t0], %[rt]")
        emit("s_cmp_ge_i32 %[t0], 0")
        emit("s_cbranch_scc1 2f")
        emit("v_readfirstlane_b32 %[t0], %[vq]")
        emit("s_cmp_lg_u32 %[t0], 0")
        emit("s_mov_b32 %[st], 1")
        emit("s_cbranch_scc1 9f")
        emit("s_add_u32 %[spins], %[spins], 1")
        emit("s_cmp_gt_i32 %[spins], %[lim]")
        emit("s_mov_b32 %[st], 2")
        emit("s_cbranch_scc1 9f")
        emit("s_sleep 1")
        emit("s_branch 3b")
        emit("2:")
        emit("s_mov_b32 %[st], 0")

    def enter(site, u):
        # the read stream moves on to K-iteration u > 0: check its slot is
        # full, move both addresses by the slot's byte delta, peek at u + 1
        next_slot("rs", "rt", "t0")
        check(site, u)
        emit("s_mov_b32 %[t0], %[rb]")
        emit("s_mul_i32 %%[rb], %%[rs], %d" % c.stage)
        emit("s_add_u32 %[rb], %[rb], %[ring]")
        emit("s_sub_u32 %[t0], %[rb], %[t0]")
        emit("v_add_u32 %[va], %[t0], %[va]")
        emit("v_add_u32 %[vb], %[t0], %[vb]")
        peek(u + 1)

    def release(site, u):
        E.wait_for(site, lambda tag: tag[0] in ("A", "B") and tag[1] // KS == u)
        emit("s_lshl_b32 %[t1], %[rel], 2")
        emit("s_add_u32 %[t1], %[t1], %[emptyb]")
        emit("v_mov_b32 %[vx], %[t1]")
        emit("v_mov_b32 %[vq], 1")
        emit("s_mov_b64 %[sav], exec")
        emit("s_mov_b64 exec, 1")
        E.op("ds_add_u32 %[vx], %[vq]", ("rel", u))
        emit("s_mov_b64 exec, %[sav]")
        emit("s_add_u32 %[rel], %[rel], 1")
        emit("s_cmp_eq_u32 %[rel], %[P]")
        emit("s_cselect_b32 %[rel], 0, %[rel]")

    def delay():
        emit("s_cmp_le_i32 %[dly], 0")
        emit("s_cbranch_scc1 6f")
        emit("s_mov_b32 %[t0], %[dly]")
        emit("5:")
        emit("s_sleep 127")
        emit("s_sub_u32 %[t0], %[t0], 1")
        emit("s_cmp_lg_u32 %[t0], 0")
        emit("s_cbranch_scc1 5b")
        emit("6:")

    def stamp(ev, ahead_of_ti):
        # store the low 32 bits of the shader clock as event ev of record
        # ti + ahead_of_ti (skipped past the buffer's records), from lane 0
        if not traced:
            return
        emit("s_memtime s[100:101]")
        E.emit("s_waitcnt lgkmcnt(0)")
        E.ops.clear()  # everything issued so far has completed
        emit("s_add_u32 %%[t0], %%[ti], %d" % ahead_of_ti)
        emit("s_cmp_lt_u32 %[t0], %[tlim]")
        emit("s_cbranch_scc0 7f")
        emit("s_lshl_b32 %[t1], %[t0], 5")
        emit("s_add_u32 %%[t1], %%[t1], %d" % (4 * ev))
        emit("v_mov_b32 %[vx], %[t1]")
        emit("v_mov_b32 %[vq], s100")
        emit("s_mov_b64 %[sav], exec")
        emit("s_mov_b64 exec, 1")
        emit("global_store_dword %[vx], %[vq], %[tr]")
        emit("s_mov_b64 exec, %[sav]")
        emit("s_nop 1")
        emit("7:")

    def kstep(seg, t, ahead):
        # k-step t of the tile; ahead: k-step t + 1 exists (read it now)
        kss = t % KS
        last_of_iter = kss == KS - 1
        if traced and kss == 0:
            emit("s_add_u32 %[ti], %[ti], 1")  # K-iteration t / KS of the tile starts
        for mb in range(c.bm):
            E.wait_for((seg, kss, "a", mb), lambda tag, mb=mb: tag == ("A", t, mb) or
                       (mb == 0 and tag == ("B", t, 0)))
            mf(mb, 0)
        if kss == 0:
            stamp(5, 0)
        if ahead and last_of_iter:
            enter((seg, kss, "enter"), (t + 1) // KS)
            stamp(4, 1)
        if ahead:
            read_b(t + 1, 0)
        E.wait_for((seg, kss, "b1"), lambda tag: tag == ("B", t, 1))
        mf(0, 1)
        if last_of_iter:
            release((seg, kss, "rel"), t // KS)
            stamp(6, 0)
        if ahead:
            emit("v_xor_b32 %%[va], %d, %%[va]" % _kxor(kss, (t + 1) % KS))
            read_a(t + 1, 0)
        for mb in range(1, c.bm):
            mf(mb, 1)
            if ahead:
                read_a(t + 1, mb)
        if ahead:
            read_b(t + 1, 1)

    # entry: the caller has waited for the tile's first slot (slot, ft) and
    # pointed va / vb at k-step 0 of it; the accumulators were just written by
    # VALU instructions
    emit("s_nop 7")
    emit("s_mov_b32 %[st], 0")
    emit("s_mov_b32 %[rs], %[slot]")
    emit("s_mov_b32 %[rt], %[ft]")
    emit("s_mov_b32 %[rel], %[slot]")
    if traced:
        emit("s_sub_u32 %[ti], %[tq], 1")  # record index of the K-iteration under way
    emit("s_mul_i32 %%[rb], %%[rs], %d" % c.stage)
    emit("s_add_u32 %[rb], %[rb], %[ring]")
    peek(1)
    # prologue: the reads of k-step 0, in the order the loop issues them
    read_b(0, 0)
    for mb in range(c.bm):
        read_a(0, mb)
    read_b(0, 1)
    # S - 1 loop bodies (one K-iteration each, the last k-step entering the
    # next slot), then the tile's last K-iteration
    emit("s_sub_u32 %[kk], %[S], 1")
    emit("s_cmp_eq_u32 %[kk], 0")
    emit("s_cbranch_scc1 8f")
    emit("1:")
    for u in range((S - 1) if S is not None else 1):
        delay()
        for j in range(KS):
            kstep("body", u * KS + j, True)
    emit("s_sub_u32 %[kk], %[kk], 1")
    emit("s_cmp_lg_u32 %[kk], 0")
    emit("s_cbranch_scc1 1b")
    emit("8:")
    delay()
    u_last = (S - 1) if S is not None else 0
    for j in range(KS):
        kstep("tail", u_last * KS + j, j < KS - 1)
    # hand back the slot and target of the next tile's first K-iteration
    next_slot("rs", "rt", "t0")
    emit("s_mov_b32 %[slot], %[rs]")
    emit("s_mov_b32 %[ft], %[rt]")
    emit("9:")
    # nothing of this block may still be in flight (the peek of the next
    # tile's counter, or reads left by an abort), and the caller reads the
    # accumulators with VALU instructions
    emit("s_waitcnt lgkmcnt(0)")
    for _ in range(3):
        emit("s_nop 15")


def gen_roll_block(c: RollCfg, bf16: bool, traced: bool = False) -> list[str]:
    waits = {}
    for S in (1, 2, 3, 5):
        E = Emitter()
        program_roll(E, c, bf16, S, traced)
        for site, n in E.need.items():
            waits[site] = min(waits.get(site, LGKM_MAX), n)
    E = Emitter(waits)
    program_roll(E, c, bf16, None, traced)
    return E.lines


_ROLL_FN = """  static __device__ __forceinline__ uint32_t %(name)s(f32x16_t (&c)[%(bm)d][%(bn)d], uint32_t va, uint32_t vb,
                                                  uint32_t& slot, uint32_t& ftarget, uint32_t P, uint32_t S,
                                                  uint32_t ring, uint32_t fullb, uint32_t emptyb, uint32_t abortb,
                                                  int32_t lim, int32_t dly%(targs)s) {
#if defined(__HIP_DEVICE_COMPILE__)
    uint32_t st, rs, rt, rb, rel, kk, t0, t1, spins, vp, vq, vx%(tvars)s;
    uint64_t sav;
    asm volatile(
%(body)s
        : %(acc)s, [slot] "+s"(slot), [ft] "+s"(ftarget), [st] "=&s"(st), [rs] "=&s"(rs), [rt] "=&s"(rt),
          [rb] "=&s"(rb), [rel] "=&s"(rel), [kk] "=&s"(kk), [t0] "=&s"(t0), [t1] "=&s"(t1),
          [spins] "=&s"(spins), [sav] "=&s"(sav), [va] "+v"(va), [vb] "+v"(vb), [vp] "=&v"(vp),
          [vq] "=&v"(vq), [vx] "=&v"(vx)%(touts)s
        : [P] "s"(P), [S] "s"(S), [ring] "s"(ring), [fullb] "s"(fullb), [emptyb] "s"(emptyb),
          [abortb] "s"(abortb), [lim] "s"(lim), [dly] "s"(dly)%(tins)s
        : "memory", "scc", %(clobbers)s%(tclob)s);
    return st;
#else
    (void)c; (void)va; (void)vb; (void)slot; (void)ftarget; (void)P; (void)S; (void)ring;
    (void)fullb; (void)emptyb; (void)abortb; (void)lim; (void)dly;%(tvoid)s
    return 0;
#endif
  }
"""


def gen_roll_struct(c: RollCfg, bf16: bool) -> str:
    acc_ops = ", ".join('[c%d_%d] "+v"(c[%d][%d])' % (mb, nb, mb, nb) for mb in range(c.bm) for nb in range(c.bn))
    clobbers = ", ".join('"v%d"' % r for r in range(c.frag_base, c.vgprs))
    fns = []
    for traced in (False, True):
        lines = gen_roll_block(c, bf16, traced)
        body = "\n".join('        "%s\\n\\t"' % l for l in lines)
        t = dict(targs="", tvars="", touts="", tins="", tclob="", tvoid="")
        if traced:
            t = dict(targs=",\n                                                  uint32_t* trace, uint32_t tq, uint32_t tlim",
                     tvars=", ti", touts=', [ti] "=&s"(ti)',
                     tins=', [tr] "s"(trace), [tq] "s"(tq), [tlim] "s"(tlim)', tclob=', "s100", "s101"',
                     tvoid=" (void)trace; (void)tq; (void)tlim;")
        fns.append(_ROLL_FN % dict(name="tile_traced" if traced else "tile", bm=c.bm, bn=c.bn, body=body,
                                   acc=acc_ops, clobbers=clobbers, **t))
    return """template <>
struct RollLoop<%(tm)d, %(tn)d, %(tk)d, %(nc)d, %(np)d, %(bf16)s> {
  static constexpr bool kAvailable = true;
  // va / vb: this lane's A and B read addresses for k-step 0 of the tile's
  // first slot (moved along by the block).  tile_traced also stores the
  // consumer's event stamps of K-iterations tq, tq + 1, ... of the trace
  // record buffer `trace` (tlim records).
%(fns)s};
""" % dict(tm=c.tm, tn=c.tn, tk=c.tk, nc=c.nc, np=c.np, bf16="true" if bf16 else "false",
           fns="\n".join(fns))


def generate() -> str:
    parts = ["// generated by paper_2506_11209_amd/csrc/gen_deep_loop.py -- do not edit",
             "// The K loop of one output tile for the deep-prefetch consumer (consumer_deep",
             "// in ws_gemm_kernel.hpp), one asm block per kernel configuration.",
             "",
             "template <int TM, int TN, int TK, int NC, int NP, bool BF16>",
             "struct DeepLoop {",
             "  static constexpr bool kAvailable = false;",
             "  static constexpr int kIterQuantum = 1;",
             "};",
             ""]
    for t in CONFIGS:
        for bf16 in (True, False):
            parts.append(gen_struct(Cfg(*t), bf16))
    parts += ["// The K loop of one output tile for two consumer waves per SIMD (consumer_roll).",
              "template <int TM, int TN, int TK, int NC, int NP, bool BF16>",
              "struct RollLoop {",
              "  static constexpr bool kAvailable = false;",
              "};",
              ""]
    for t in ROLL_CONFIGS:
        for bf16 in (True, False):
            parts.append(gen_roll_struct(RollCfg(*t), bf16))
    return "\n".join(parts)


def main(argv=None):
    argv = sys.argv[1:] if argv is None else argv
    text = generate()
    if "--check" in argv:
        with open(OUT) as f:
            same = f.read() == text
        print("ws_deep_loop.inc is %s" % ("up to date" if same else "STALE"))
        return 0 if same else 1
    with open(OUT, "w") as f:
        f.write(text)
    print("wrote", OUT)
    return 0


if __name__ == "__main__":
    sys.exit(main())
