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
every LDS wait is placed by hand.  The schedule and its wait counts are
explained in ws_gemm_kernel.hpp (consumer_deep).

A K-iteration has four k-steps (TK = 64, one 32x32x16 MFMA per 32x32 block
and k-step).  Fragment set s (k-step s of a slot) holds BM A fragments
(ds_read_b128) and BN B fragments (two ds_read_b64_tr_b16 each).
"""
from __future__ import annotations

import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
OUT = os.path.join(HERE, "ws_deep_loop.inc")

# (TM, TN, TK, NC, SPLIT): the configurations that get the deep consumer
# (four consumer waves in a 2 x 2 grid, one producer group, TK = 64).
CONFIGS = [(256, 128, 64, 4, 1), (128, 256, 64, 4, 1), (128, 128, 64, 4, 1)]
HEADER_BYTES = 256


class Cfg:
    def __init__(self, tm, tn, tk, nc, split):
        assert nc == 4 and split == 1 and tk == 64
        self.tm, self.tn, self.tk, self.nc, self.split = tm, tn, tk, nc, split
        self.np = nc * split
        self.wm, self.wn = tm // 2, tn // 2
        self.bm, self.bn = self.wm // 32, self.wn // 32
        self.nq = tn // 16
        self.a_bytes = tm * tk * 2
        self.stage = self.a_bytes + tk * tn * 2
        self.reads = self.bm + 2 * self.bn            # LDS instructions per fragment set
        self.set_regs = 4 * (self.bm + self.bn)
        self.frag_base = 256 - 4 * self.set_regs      # four sets at the top of the file
        assert self.reads <= 15 and self.bm * self.bn * 16 + 4 * self.set_regs <= 224
        assert self.stage % 128 == 0 and HEADER_BYTES % 128 == 0


def gen_block(c: Cfg, bf16: bool) -> list[str]:
    """Lines of the asm program (operands by name)."""
    mfma = "v_mfma_f32_32x32x16_bf16" if bf16 else "v_mfma_f32_32x32x16_f16"
    w2r = min(15, 2 * c.reads)
    w2r2 = min(15, 2 * c.reads + 2)
    out = []
    emit = out.append

    def a_reg(s, mb):
        b = c.frag_base + s * c.set_regs + 4 * mb
        return "v[%d:%d]" % (b, b + 3)

    def b_regs(s, nb):
        b = c.frag_base + s * c.set_regs + 4 * c.bm + 4 * nb
        return "v[%d:%d]" % (b, b + 3), "v[%d:%d]" % (b, b + 1), "v[%d:%d]" % (b + 2, b + 3)

    def addr(s, base):
        # the two address registers of fragment set s in the slot at SGPR `base`
        emit("v_add_u32 %%[va], %%[%s], %%[aoff]" % base)
        if s:
            emit("v_xor_b32 %%[va], %d, %%[va]" % (32 * s))
        emit("v_add_u32 %%[vb], %%[%s], %%[boff]" % base)

    def reads(s):
        out = []
        for mb in range(c.bm):
            off = mb * 32 * c.tk * 2
            assert off < 65536
            out.append("ds_read_b128 %s, %%[va] offset:%d" % (a_reg(s, mb), off))
        for nb in range(c.bn):
            _, lo, hi = b_regs(s, nb)
            off = ((4 * s) * c.nq + 2 * nb) * 128
            assert off + c.nq * 128 < 65536
            out.append("ds_read_b64_tr_b16 %s, %%[vb] offset:%d" % (lo, off))
            out.append("ds_read_b64_tr_b16 %s, %%[vb] offset:%d" % (hi, off + c.nq * 128))
        return out

    def mfma_list(s):
        out = []
        for mb in range(c.bm):
            for nb in range(c.bn):
                full, _, _ = b_regs(s, nb)
                out.append("%s %%[c%d_%d], %s, %s, %%[c%d_%d]" % (mfma, mb, nb, a_reg(s, mb), full, mb, nb))
        return out

    def issue(s, base):
        addr(s, base)
        for l in reads(s):
            emit(l)

    def mfmas(s):
        for l in mfma_list(s):
            emit(l)

    def step(s_mfma, s_read, base):
        # the MFMAs of set s_mfma with the reads of set s_read (in the slot at
        # `base`) between them: read, MFMA, read, MFMA, ...  A wave tracks at
        # most 15 LDS operations, so a read can stall at issue; one MFMA after
        # each keeps the matrix core fed meanwhile (measured faster than
        # issuing a set's reads together, before or after its MFMAs).
        addr(s_read, base)
        ms, rs = mfma_list(s_mfma), reads(s_read)
        while ms or rs:
            if rs:
                emit(rs.pop(0))
            if ms:
                emit(ms.pop(0))

    def wait(n):
        emit("s_waitcnt lgkmcnt(%d)" % n)

    def slot_base(dst, slot):
        emit("s_mul_i32 %%[%s], %%[%s], %d" % (dst, slot, c.stage))
        emit("s_add_u32 %%[%s], %%[%s], %%[ring]" % (dst, dst))

    def next_slot():
        # (ns, nt) <- the slot and full-counter target of the K-iteration after (slot, ft)
        emit("s_add_u32 %[ns], %[slot], 1")
        emit("s_add_u32 %%[t0], %%[ft], %d" % c.np)
        emit("s_cmp_eq_u32 %[ns], %[P]")
        emit("s_cselect_b32 %[ns], 0, %[ns]")
        emit("s_cselect_b32 %[nt], %[t0], %[ft]")

    def peek(slot_reg, wrap_next):
        # issue a read of full[slot] (full[next(slot)] when wrap_next) into vp
        if wrap_next:
            emit("s_add_u32 %%[t1], %%[%s], 1" % slot_reg)
            emit("s_cmp_eq_u32 %[t1], %[P]")
            emit("s_cselect_b32 %[t1], 0, %[t1]")
            emit("s_lshl_b32 %[t1], %[t1], 2")
        else:
            emit("s_lshl_b32 %%[t1], %%[%s], 2" % slot_reg)
        emit("s_add_u32 %[t1], %[t1], %[fullb]")
        emit("v_mov_b32 %[vx], %[t1]")
        emit("ds_read_b32 %[vp], %[vx]")

    def release(n):
        # one ds_add from lane 0 once at most n younger LDS operations are outstanding
        emit("s_lshl_b32 %[t1], %[slot], 2")
        emit("s_add_u32 %[t1], %[t1], %[emptyb]")
        emit("v_mov_b32 %[vx], %[t1]")
        emit("v_mov_b32 %[vq], 1")
        wait(n)
        emit("s_mov_b64 %[sav], exec")
        emit("s_mov_b64 exec, 1")
        emit("ds_add_u32 %[vx], %[vq]")
        emit("s_mov_b64 exec, %[sav]")

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

    def check_next():
        # vp holds full[ns] as peeked; spin (draining every read) only when short
        emit("v_readfirstlane_b32 %[t0], %[vp]")
        emit("s_sub_u32 %[t0], %[t0], %[nt]")
        emit("s_cmp_ge_i32 %[t0], 0")
        emit("s_cbranch_scc1 2f")
        emit("s_mov_b32 %[spins], 0")
        emit("s_lshl_b32 %[t1], %[ns], 2")
        emit("s_add_u32 %[t1], %[t1], %[fullb]")
        emit("3:")
        emit("v_mov_b32 %[vx], %[t1]")
        emit("ds_read_b32 %[vp], %[vx]")
        emit("v_mov_b32 %[vx], %[abortb]")
        emit("ds_read_b32 %[vq], %[vx]")
        wait(0)
        emit("v_readfirstlane_b32 %[t0], %[vp]")
        emit("s_sub_u32 %[t0], %[t0], %[nt]")
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
        emit("s_mov_b32 %[st], 0")  # the poll may have set it before a branch not taken

    # entry: the caller has waited for the first slot of the tile; the
    # accumulators were just written by VALU instructions
    emit("s_nop 7")
    emit("s_mov_b32 %[st], 0")
    slot_base("base", "slot")
    next_slot()
    issue(0, "base")
    issue(1, "base")
    emit("s_cmp_gt_u32 %[S], 1")
    emit("s_cbranch_scc0 4f")
    peek("ns", False)
    emit("4:")
    issue(2, "base")
    emit("s_sub_u32 %[kk], %[S], 1")
    emit("s_cmp_eq_u32 %[kk], 0")
    emit("s_cbranch_scc1 8f")
    # steady K-iteration (the next one is in the same tile)
    emit("1:")
    delay()
    wait(w2r)
    step(0, 3, "base")
    wait(w2r)
    check_next()
    slot_base("nbase", "ns")
    step(1, 0, "nbase")
    wait(w2r)
    step(2, 1, "nbase")
    release(w2r)
    peek("ns", True)
    wait(w2r2)
    step(3, 2, "nbase")
    emit("s_mov_b32 %[slot], %[ns]")
    emit("s_mov_b32 %[ft], %[nt]")
    emit("s_mov_b32 %[base], %[nbase]")
    next_slot()
    emit("s_sub_u32 %[kk], %[kk], 1")
    emit("s_cmp_lg_u32 %[kk], 0")
    emit("s_cbranch_scc1 1b")
    # last K-iteration of the tile: nothing is read ahead
    emit("8:")
    delay()
    wait(w2r)
    step(0, 3, "base")
    wait(w2r)
    mfmas(1)
    wait(c.reads)
    mfmas(2)
    release(0)
    mfmas(3)
    emit("s_mov_b32 %[slot], %[ns]")
    emit("s_mov_b32 %[ft], %[nt]")
    emit("9:")
    # the caller reads the accumulators with VALU instructions
    for _ in range(3):
        emit("s_nop 15")
    return out


def gen_struct(c: Cfg, bf16: bool) -> str:
    lines = gen_block(c, bf16)
    acc_ops = ", ".join('[c%d_%d] "+v"(c[%d][%d])' % (mb, nb, mb, nb) for mb in range(c.bm) for nb in range(c.bn))
    clobbers = ", ".join('"v%d"' % r for r in range(c.frag_base, 256))
    body = "\n".join('        "%s\\n\\t"' % l if not l.endswith(":") else '        "%s\\n\\t"' % l for l in lines)
    return """template <>
struct DeepLoop<%(tm)d, %(tn)d, %(tk)d, %(nc)d, %(split)d, %(bf16)s> {
  static constexpr bool kAvailable = true;
  static __device__ __forceinline__ uint32_t tile(f32x16_t (&c)[%(bm)d][%(bn)d], uint32_t a_off0, uint32_t b_off,
                                                  uint32_t& slot, uint32_t& ftarget, uint32_t P, uint32_t S,
                                                  uint32_t ring, uint32_t fullb, uint32_t emptyb, uint32_t abortb,
                                                  int32_t lim, int32_t dly) {
#if defined(__HIP_DEVICE_COMPILE__)
    uint32_t st, ns, nt, kk, base, nbase, t0, t1, spins, va, vb, vp, vq, vx;
    uint64_t sav;
    asm volatile(
%(body)s
        : %(acc)s, [slot] "+s"(slot), [ft] "+s"(ftarget), [st] "=&s"(st), [ns] "=&s"(ns), [nt] "=&s"(nt),
          [kk] "=&s"(kk), [base] "=&s"(base), [nbase] "=&s"(nbase), [t0] "=&s"(t0), [t1] "=&s"(t1),
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
""" % dict(tm=c.tm, tn=c.tn, tk=c.tk, nc=c.nc, split=c.split, bf16="true" if bf16 else "false", bm=c.bm,
           bn=c.bn, body=body, acc=acc_ops, clobbers=clobbers)


def generate() -> str:
    parts = ["// generated by paper_2506_11209_amd/csrc/gen_deep_loop.py -- do not edit",
             "// The K loop of one output tile for the deep-prefetch consumer (consumer_deep",
             "// in ws_gemm_kernel.hpp), one asm block per kernel configuration.",
             "",
             "template <int TM, int TN, int TK, int NC, int SPLIT, bool BF16>",
             "struct DeepLoop {",
             "  static constexpr bool kAvailable = false;",
             "};",
             ""]
    for t in CONFIGS:
        for bf16 in (True, False):
            parts.append(gen_struct(Cfg(*t), bf16))
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
