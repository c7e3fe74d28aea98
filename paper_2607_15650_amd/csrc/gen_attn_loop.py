"""Writes attn_d128_loop.inc and attn_d64_loop.inc: the key loop of the bf16
attention kernel at head dim 128 and 64 as one block of gfx950 assembly
each, scheduled by hand.

The loop computes, for one task (256 query rows of one head against the keys
of one partition), the unnormalised attention state of Sec. 2.2.4
(Eq. attention_state) by online softmax: O^T = sum over key tiles of V^T P^T
with P = exp2(scale*log2(e)*K Q^T - m), the running maximum m and the
per-lane row sums.  The arithmetic is the same as the compiled kernels'; what
the hand schedule adds is register placement and instruction order:

  * one wave per SIMD (4 waves, 256 rows), each with two 32-row query blocks,
    so that every K or V^T fragment read from LDS feeds two MFMAs;
  * Q^T fragments and the O^T accumulators live in AGPRs (a128-a191,
    a0-a127); scores, probabilities and the rest in VGPRs;
  * each 64-key iteration is 32 fragment steps of two MFMAs: scores of tile
    i+1 (16 steps) beside the exponentials of the second half of tile i, then
    P V of tile i (16 steps) beside the exponentials of the first half of
    tile i+1; every MFMA gap carries about one exp2, one FMA, one add and half
    a bf16 conversion;
  * the LDS fragment reads form one stream, LA steps ahead, across the groups
    of an iteration and into the next iteration, so the matrix core does not
    wait for a fragment where one group of MFMAs hands over to the next;
  * K and V tiles go into a 4-deep LDS ring with buffer loads that write LDS
    directly; the buffer descriptor ends at the partition's last key, so rows
    past the end read as zeros without touching memory; every wave issues
    its quarter of a tile pair one 1 KiB load at a time, spread over the
    steps before the barrier, with one m0 per tile and the loads of a tile
    at immediate offsets of 1 KiB (the offset moves both the global and the
    LDS address, and the range check includes it);
  * the steady loop takes no branch but its loop-back: iterations run in
    blocks of four while none of the four is the last or masks a partial
    last tile, and the tests for those two run only in the few iterations
    after the blocks; the tail mask is out of line;
  * two forms of the block: the checked one tests every tile's sums for the
    lazy maximum and branches out of line into the slow path that raises
    m; the fast one takes m from tile 0's scores in the prologue and never
    raises it (no test, no branch per tile).  The kernel runs the fast form
    and runs a task again in the checked form when a row sum ends above
    2^40 or NaN; below that bound no tile of the checked form would have
    raised m, so the two agree bit for bit.

Register and LDS layout, the lazy running maximum and the accumulator layout
of the 32x32x16 MFMA follow attn_bf16.hip.  Run `python gen_attn_loop.py`
in this directory after editing; the build compiles the .inc as written.
"""
from __future__ import annotations

import os
import sys

# ---------------------------------------------------------------- registers
def S(par, kb, qb):            # scores, 16 VGPRs: parity par, key block kb, query block qb
    return 64 * par + 32 * kb + 16 * qb


def P(par, kb, qb, hh):        # bf16 probabilities, 4 VGPRs (8 keys)
    return 128 + 32 * par + 16 * kb + 8 * qb + 4 * hh


NFRAG = 8                      # fragment buffers (32 steps per iteration)
LA = 6                         # fragment reads issued this many steps ahead
WAITK = 4                      # one LDS wait per this many steps


def FRAG(f):
    return 192 + 4 * (f % NFRAG)


TMP = 224                      # 4 VGPRs: the exponentials in flight


def T(qb):                     # tile row sums (this lane's keys)
    return 228 + qb


def M(qb):                     # running maximum (log2 units)
    return 230 + qb


def L(qb):                     # row sums (this lane's keys)
    return 232 + qb


def KADDR(s):                  # LDS byte address of this lane's K fragment, k-step s
    return 234 + s


def VADDR(db):                 # LDS byte address of this lane's V^T transpose reads, dim block db
    return 234 + KS + db


def DMAK(j):                   # byte offset of this lane's 16 bytes in a K tile, load j
    return 234 + KS + DB + j


def DMAV(j):
    return 234 + KS + DB + LW + j


QPTR = 64                      # v[64:67]: the lane's Q row addresses, one per query block


def O(qb, db):                 # AGPR accumulators of O^T
    return 16 * DB * qb + 16 * db


def Q(qb, s):                  # AGPR Q^T fragments
    return 128 + 32 * qb + 4 * s


# scalar registers: inputs pinned by the caller, then scratch
S_SL2, S_NT, S_KVLEN, S_WLDS, S_TILEB = 40, 41, 42, 44, 45
S_KD, S_VD = 48, 52            # buffer descriptors (4 each)
S_I, S_TMP, S_BIG, S_MASKAT, S_RET, S_CMP, S_NTM1, S_LIM = 56, 57, 58, 59, 60, 62, 64, 65
SCRATCH_SGPRS = list(range(56, 66))

KRING = 0                      # LDS byte offset of the K ring


def configure(d):
    """Head dimension d (128 or 64): k-steps and dim blocks of the MFMAs, tile
    bytes, 1 KiB loads per wave per tile, the V ring's offset, and where in
    the iteration's steps the tile loads and the barrier sit."""
    global D, KS, DB, ROWB, TILEB, LW, VRING, NQ, NP, LOAD_STEP, BARRIER_STEP
    D = d
    KS, DB = d // 16, d // 32
    ROWB = 2 * d                   # bytes per key row
    TILEB = 64 * ROWB              # 64-key tile
    LW = TILEB // 1024 // 4        # 1 KiB loads per wave per tile
    VRING = 4 * TILEB              # the V ring follows the K ring (VADDR includes it)
    NQ, NP = 2 * KS, 4 * DB        # score steps, P V steps
    # the barrier that publishes the next tiles comes before the first read
    # of the next iteration's K tile (issued LA steps before its step, right
    # behind the first MFMA of a step, ahead of that step's events)
    BARRIER_STEP = min(3 * (NQ + NP) // 4, NQ + NP - LA - 1)
    # the wave's 2 LW loads of an iteration (K, then V), one per step, spread
    # over the steps before the barrier (measured: one load per event beats
    # two or four, and branching to a per-wave burst cost about 8 % of the
    # loop's cycles)
    LOAD_STEP = [k * BARRIER_STEP // (2 * LW) for k in range(2 * LW)]
    assert NQ + NP - LA > BARRIER_STEP and LOAD_STEP[-1] < BARRIER_STEP
    assert len(set(LOAD_STEP)) == 2 * LW


configure(128)


def kslot(t):
    return KRING + (t % 4) * TILEB


def vslot(t):
    return (t % 4) * TILEB     # relative to VADDR


def v(a, n=1):
    return f"v{a}" if n == 1 else f"v[{a}:{a + n - 1}]"


def a_(a, n=1):
    return f"a{a}" if n == 1 else f"a[{a}:{a + n - 1}]"


def s_(a, n=1):
    return f"s{a}" if n == 1 else f"s[{a}:{a + n - 1}]"


# ---------------------------------------------------------------- softmax
def sm_ops(par, kb, qb, first):
    """exp2(s*sl2 - m) of the 16 scores of one key block and query block,
    software pipelined (FMA of e, exp2 of e-1, sum and bf16 pair of e-2),
    the row sum into T(qb); `first`: the tile's first block, which starts T"""
    ops = []
    base = S(par, kb, qb)
    for step in range(18):
        e = step
        if e < 16:
            ops.append(f"v_fma_f32 {v(TMP + e % 4)}, {v(base + e)}, {s_(S_SL2)}, -{v(M(qb))}")
        e = step - 1
        if 0 <= e < 16:
            ops.append(f"v_exp_f32 {v(TMP + e % 4)}, {v(TMP + e % 4)}")
        e = step - 2
        if 0 <= e < 16:
            if first and e == 0:
                ops.append(f"v_mov_b32 {v(T(qb))}, {v(TMP + e % 4)}")
            else:
                ops.append(f"v_add_f32 {v(T(qb))}, {v(T(qb))}, {v(TMP + e % 4)}")
            if e % 2 == 1:
                hh, j = e // 8, (e % 8) // 2
                ops.append(f"v_cvt_pk_bf16_f32 {v(P(par, kb, qb, hh) + j)}, {v(TMP + (e - 1) % 4)}, {v(TMP + e % 4)}")
    return ops


# ---------------------------------------------------------------- steps
class Step:
    """one fragment: its LDS reads and the two MFMAs that consume it"""
    def __init__(self, reads, mfmas):
        self.reads = reads
        self.mfmas = mfmas


def qk_steps(nxt, t_next, buf0=0):
    """scores of tile t_next into S(nxt): 16 steps, k-step s outer, key block
    kb inner (an accumulator is reused every fourth MFMA)"""
    out = []
    for s in range(KS):
        for kb in range(2):
            f = buf0 + 2 * s + kb
            rd = [f"ds_read_b128 {v(FRAG(f), 4)}, {v(KADDR(s))} offset:{kslot(t_next) + kb * 32 * ROWB}"]
            mf = []
            for qb in range(2):
                src_c = "0" if s == 0 else v(S(nxt, kb, qb), 16)
                mf.append(f"v_mfma_f32_32x32x16_bf16 {v(S(nxt, kb, qb), 16)}, {v(FRAG(f), 4)}, {a_(Q(qb, s), 4)}, {src_c}")
            out.append(Step(rd, mf))
    return out


def pv_steps(cur, t_cur, buf0=None):
    """O^T += V^T P^T over tile t_cur: 16 steps, key block kb, 16-key step s,
    dim block db (an accumulator is reused every eighth MFMA)"""
    out = []
    k = 0
    buf0 = NQ if buf0 is None else buf0
    for kb in range(2):
        for s in (2 * kb, 2 * kb + 1):
            for db in range(DB):
                f = buf0 + k
                k += 1
                off = vslot(t_cur) + 16 * s * ROWB
                rd = [f"ds_read_b64_tr_b16 {v(FRAG(f), 2)}, {v(VADDR(db))} offset:{off}",
                      f"ds_read_b64_tr_b16 {v(FRAG(f) + 2, 2)}, {v(VADDR(db))} offset:{off + 8 * ROWB}"]
                mf = [f"v_mfma_f32_32x32x16_bf16 {a_(O(qb, db), 16)}, {v(FRAG(f), 4)}, {v(P(cur, kb, qb, s % 2), 4)}, {a_(O(qb, db), 16)}"
                      for qb in range(2)]
                out.append(Step(rd, mf))
    return out


def stream(steps, nxt_steps, valu_by_step, events, issued, pre_events=None):
    """Emits the steps' MFMAs with their fragment reads LA steps ahead
    (continuing into nxt_steps, whose reads are issued but not consumed),
    the VALU ops of each step spread after its two MFMAs, and events
    (instruction lists) at given step indices: `pre_events` before the
    step's wait and MFMAs (code that the step's MFMAs depend on), `events`
    behind its first MFMA.  `issued`: how many of the first steps' reads the
    code before has already issued.

    Order within a step (measured, 64-key iterations on the video-DiT
    workload): one LDS wait per WAITK steps, covering them all; the step's
    first MFMA; the first read of step f+LA; the step's events; half the
    VALU ops; the second MFMA; the other read(s) of step f+LA; the other
    VALU ops.  Reads issued right behind an MFMA cost least: placed before
    the wait the loop took 11 % longer, after a VALU op 12 % longer."""
    out = []
    allst = steps + nxt_steps
    n = len(steps)
    nissued = issued              # steps [0, nissued) of allst have their reads issued

    def issue_upto(k):
        nonlocal nissued
        while nissued <= k and nissued < len(allst):
            out.extend(allst[nissued].reads)
            nissued += 1

    issue_upto(LA - 1)
    pre_events = pre_events or {}
    for f in range(n):
        out.extend(pre_events.get(f, []))
        if f % WAITK == 0:
            upto = min(f + WAITK - 1, n - 1, nissued - 1)
            later = sum(len(allst[j].reads) for j in range(upto + 1, nissued))
            out.append(f"s_waitcnt lgkmcnt({later})")
        valu = valu_by_step.get(f, [])
        half = (len(valu) + 1) // 2
        k = f + LA
        rd = allst[k].reads if nissued == k and k < len(allst) else []
        out.append(steps[f].mfmas[0])
        out.extend(rd[:1])
        out.extend(events.get(f, []))
        out.extend(valu[:half])
        out.append(steps[f].mfmas[1])
        out.extend(rd[1:])
        if rd:
            nissued = k + 1
        out.extend(valu[half:])
    out.extend(events.get(n, []))
    return out


def spread_valu(ops, first_step, nsteps):
    """assigns a list of VALU ops evenly to nsteps consecutive steps"""
    res = {}
    per = len(ops) / nsteps
    vi = 0
    for k in range(nsteps):
        hi = len(ops) if k == nsteps - 1 else round(per * (k + 1))
        res[first_step + k] = ops[vi:hi]
        vi = hi
    return res


# ---------------------------------------------------------------- loads
def dma_tile(desc, ring_off, t):
    """this wave's LW 1 KiB loads of a tile into ring slot t % 4, one list of
    instructions per load: m0 is set to the wave's first KiB of the slot once,
    and load j adds j KiB through its immediate offset, which moves the LDS
    destination and the global address alike (the lane's offset register
    holds its byte offset minus j KiB)"""
    base = DMAK if desc == S_KD else DMAV
    out = [[f"s_add_u32 m0, {s_(S_WLDS)}, {ring_off + (t % 4) * TILEB}", "s_nop 0"]]
    for j in range(LW):
        off = f" offset:{1024 * j}" if j else ""
        out[-1].append(f"buffer_load_dwordx4 {v(base(j))}, {s_(desc, 4)}, 0 offen{off} lds")
        if j + 1 < LW:
            out.append([])
    return out


def desc_advance(desc):
    """the descriptor moves on by one tile; its record count saturates at 0"""
    return [f"s_add_u32 {s_(desc)}, {s_(desc)}, {s_(S_TILEB)}",
            f"s_addc_u32 {s_(desc + 1)}, {s_(desc + 1)}, 0",
            f"s_sub_u32 {s_(desc + 2)}, {s_(desc + 2)}, {s_(S_TILEB)}",
            f"s_cselect_b32 {s_(desc + 2)}, 0, {s_(desc + 2)}"]


# ---------------------------------------------------------------- generator
class Gen:
    def __init__(self, fast=False):
        self.fast = fast          # the fast form: no per-tile test of the running maximum
        self.lines = []
        self.cold = []            # out-of-line code, emitted after the loop
        self.nlabel = 0

    @staticmethod
    def label(name):
        return f".{name}_%="

    def uniq(self, base):
        self.nlabel += 1
        return f".{base}{self.nlabel}_%="

    def call_seq(self, target):
        """instructions that branch to a block returning through s_setpc_b64"""
        pc = self.uniq("Lpc")
        ret = self.uniq("Lret")
        return [f"s_getpc_b64 {s_(S_RET, 2)}", f"{pc}:",
                f"s_add_u32 {s_(S_RET)}, {s_(S_RET)}, {ret}-{pc}",
                f"s_addc_u32 {s_(S_RET + 1)}, {s_(S_RET + 1)}, 0",
                f"s_branch {target}", f"{ret}:"]

    def out_of_line(self, cond_branch, body):
        """a conditional branch to cold code that runs body and comes back"""
        cold = self.uniq("Lcold")
        back = self.uniq("Lback")
        self.cold += [f"{cold}:"] + body + [f"s_branch {back}"]
        return [f"{cond_branch} {cold}", f"{back}:"]


def load_events(u):
    """the wave's loads of iteration u (ring phase u % 4), K_{i+3} and
    V_{i+2}, one per step of LOAD_STEP"""
    loads = dma_tile(S_KD, KRING, u + 3) + dma_tile(S_VD, VRING, u + 2)
    return {LOAD_STEP[k]: loads[k] for k in range(2 * LW)}


def check_event(g, par):
    """the lazy maximum test of tile i (parity par): a lane whose tile sum
    exceeds 2^40, or is not a number, sends the wave through the slow path;
    then the tile sums join the row sums.  The fast form only adds the tile
    sums: its maximum is tile 0's, and the kernel tests the row sums once,
    after the loop (a row sum within 2^40 bounds every tile sum of the row)."""
    if g.fast:
        return [f"v_add_f32 {v(L(0))}, {v(L(0))}, {v(T(0))}",
                f"v_add_f32 {v(L(1))}, {v(L(1))}, {v(T(1))}"]
    return ([f"v_cmp_nle_f32_e64 {s_(S_CMP, 2)}, {v(T(0))}, {s_(S_BIG)}",
             f"v_cmp_nle_f32_e64 vcc, {v(T(1))}, {s_(S_BIG)}",
             f"s_or_b64 vcc, vcc, {s_(S_CMP, 2)}"] +
            g.out_of_line("s_cbranch_vccnz", g.call_seq(g.label(f"Lslow{par}"))) +
            [f"v_add_f32 {v(L(0))}, {v(L(0))}, {v(T(0))}",
             f"v_add_f32 {v(L(1))}, {v(L(1))}, {v(T(1))}"])


def mask_event(g, nxt):
    """tile i+1 (scores in parity nxt) is the last and partial: mask its keys
    past the end (taken once per task)"""
    return ([f"s_cmp_eq_u32 {s_(S_I)}, {s_(S_MASKAT)}"] +
            g.out_of_line("s_cbranch_scc1", g.call_seq(g.label(f"Lmask{nxt}"))))


def iteration(g, u, tests=True):
    """steady iteration i (i % 4 == u): tile i+1 exists.  On entry the reads
    of its first LA steps are issued; on exit those of the next iteration.
    `tests`: the iteration may be the last steady one or the one that masks
    a partial last tile (false inside the blocks of four)."""
    cur, nxt = u % 2, 1 - u % 2
    steps = qk_steps(nxt, u + 1) + pv_steps(cur, u)
    nxt_steps = qk_steps(cur, u + 2)[:LA]           # next iteration: S parity flips
    valu = {}
    valu.update(spread_valu(sm_ops(cur, 1, 0, False), 0, NQ // 2))
    valu.update(spread_valu(sm_ops(cur, 1, 1, False), NQ // 2, NQ // 2))
    valu.update(spread_valu(sm_ops(nxt, 0, 0, True), NQ, NP // 2))
    valu.update(spread_valu(sm_ops(nxt, 0, 1, True), NQ + NP // 2, NP // 2))
    events = {}
    for k, ins in load_events(u).items():
        events.setdefault(k, []).extend(ins)
    # the test of tile i may redo its probabilities, and the mask changes
    # the scores of tile i+1: both before the first P V MFMA of tile i
    pre = {NQ: check_event(g, cur) + (mask_event(g, nxt) if tests else [])}
    # the wave's own loads of the previous tile pair have landed (only this
    # iteration's 2 LW loads may be in flight)
    events.setdefault(BARRIER_STEP, []).extend([f"s_waitcnt vmcnt({2 * LW})", "s_barrier"])
    # the iteration's scalar bookkeeping, spread over its last steps (after
    # every load), then the exit test
    n = NQ + NP
    events.setdefault(n - 4, []).extend(desc_advance(S_KD))
    events.setdefault(n - 3, []).extend(desc_advance(S_VD))
    events.setdefault(n - 2, []).extend([f"s_add_u32 {s_(S_I)}, {s_(S_I)}, 1"])
    g.lines += stream(steps, nxt_steps, valu, events, LA, pre)
    if tests:
        g.lines += [f"s_cmp_eq_u32 {s_(S_I)}, {s_(S_NTM1)}",
                    f"s_cbranch_scc1 {g.label(f'Llast{(u + 1) % 4}')}"]


def last_iteration(g, u):
    """iteration n-1: the second half of tile n-1's exponentials, its test,
    and P V; no scores of a next tile, no loads.  Reads prefetched for a next
    tile are drained first."""
    cur = u % 2
    g.lines += [f"{g.label(f'Llast{u}')}:", "s_waitcnt lgkmcnt(0)"]
    g.lines += sm_ops(cur, 1, 0, False) + sm_ops(cur, 1, 1, False)
    g.lines += check_event(g, cur)
    g.lines += [f"s_waitcnt vmcnt({2 * LW})", "s_barrier"]
    g.lines += stream(pv_steps(cur, u, 0), [], {}, {}, 0)
    g.lines += [f"s_branch {g.label('Ldone')}"]


def slow_block(g, par):
    """tile i (scores in parity par) is redone against a raised maximum: m
    rises to the tile's row maximum, O and l are rescaled, and both halves
    of the probabilities and tile sums are recomputed.  Temporaries: TMP and
    the probabilities of the other parity (free at every call site)."""
    X = P(1 - par, 0, 0, 0)       # 32 free VGPRs
    c = g.cold
    c += [f"{g.label(f'Lslow{par}')}:"]
    for qb in range(2):
        regs = [S(par, kb, qb) + r for kb in range(2) for r in range(16)]
        c.append(f"v_max_f32 {v(TMP)}, {v(regs[0])}, {v(regs[1])}")
        for r in regs[2:]:
            c.append(f"v_max_f32 {v(TMP)}, {v(TMP)}, {v(r)}")
        c += [f"v_mov_b32 {v(TMP + 1)}, {v(TMP)}",
              "s_nop 1",
              f"v_permlane32_swap_b32 {v(TMP)}, {v(TMP + 1)}",
              "s_nop 1",
              f"v_max_f32 {v(TMP)}, {v(TMP)}, {v(TMP + 1)}",
              f"v_mul_f32 {v(TMP)}, {s_(S_SL2)}, {v(TMP)}",
              f"v_max_f32 {v(TMP)}, {v(M(qb))}, {v(TMP)}",          # m_new
              f"v_sub_f32 {v(TMP + 2)}, {v(M(qb))}, {v(TMP)}",
              f"v_exp_f32 {v(TMP + 2)}, {v(TMP + 2)}",
              f"v_mov_b32 {v(TMP + 3)}, 0xff800000",
              f"v_cmp_eq_f32 vcc, {v(M(qb))}, {v(TMP + 3)}",
              f"v_cndmask_b32 {v(TMP + 2)}, {v(TMP + 2)}, 0, vcc",  # alpha (0 while m was -inf)
              f"v_mov_b32 {v(M(qb))}, {v(TMP)}",
              f"v_mul_f32 {v(L(qb))}, {v(L(qb))}, {v(TMP + 2)}"]
        for k0 in range(0, 16 * DB, 16):
            for k in range(16):
                c.append(f"v_accvgpr_read_b32 {v(X + k)}, {a_(O(qb, 0) + k0 + k)}")
            for k in range(16):
                c.append(f"v_mul_f32 {v(X + k)}, {v(X + k)}, {v(TMP + 2)}")
            for k in range(16):
                c.append(f"v_accvgpr_write_b32 {a_(O(qb, 0) + k0 + k)}, {v(X + k)}")
    for qb in range(2):
        c += sm_ops(par, 0, qb, True)
    for qb in range(2):
        c += sm_ops(par, 1, qb, False)
    c += ["s_nop 4", f"s_setpc_b64 {s_(S_RET, 2)}"]


def mask_block(g, par):
    """scores of parity par at keys >= kv_len % 64 of their tile -> -inf"""
    c = g.cold
    c += [f"{g.label(f'Lmask{par}')}:",
          f"s_and_b32 {s_(S_TMP)}, {s_(S_KVLEN)}, 63",
          f"v_mov_b32 {v(TMP)}, 0xff800000",
          f"v_mbcnt_lo_u32_b32 {v(TMP + 1)}, -1, 0",
          f"v_mbcnt_hi_u32_b32 {v(TMP + 1)}, -1, {v(TMP + 1)}",
          f"v_lshrrev_b32 {v(TMP + 1)}, 5, {v(TMP + 1)}",
          f"v_lshlrev_b32 {v(TMP + 1)}, 2, {v(TMP + 1)}"]        # 4 * (lane / 32)
    for kb in range(2):
        for r in range(16):
            cc = kb * 32 + 8 * (r // 4) + (r % 4)
            # key = cc + 4g >= rem  <=>  4g >= rem - cc
            c += [f"s_sub_i32 {s_(S_CMP)}, {s_(S_TMP)}, {cc}",
                  f"v_cmp_le_i32 vcc, {s_(S_CMP)}, {v(TMP + 1)}"]
            for qb in range(2):
                x = S(par, kb, qb) + r
                c.append(f"v_cndmask_b32 {v(x)}, {v(x)}, {v(TMP)}, vcc")
    c += ["s_nop 1", f"s_setpc_b64 {s_(S_RET, 2)}"]


def tile0_max():
    """m of each query block = scale*log2(e) times the row maximum of tile
    0's scores (both key blocks, the two lanes of a row combined), the value
    the slow path gives m at tile 0 in the checked form"""
    out = []
    for qb in range(2):
        regs = [S(0, kb, qb) + r for kb in range(2) for r in range(16)]
        out.append(f"v_max_f32 {v(TMP)}, {v(regs[0])}, {v(regs[1])}")
        for r in regs[2:]:
            out.append(f"v_max_f32 {v(TMP)}, {v(TMP)}, {v(r)}")
        out += [f"v_mov_b32 {v(TMP + 1)}, {v(TMP)}",
                "s_nop 1",
                f"v_permlane32_swap_b32 {v(TMP)}, {v(TMP + 1)}",
                "s_nop 1",
                f"v_max_f32 {v(TMP)}, {v(TMP)}, {v(TMP + 1)}",
                f"v_mul_f32 {v(TMP)}, {s_(S_SL2)}, {v(TMP)}",
                f"v_max_f32 {v(M(qb))}, {v(M(qb))}, {v(TMP)}"]
    return out + ["s_nop 2"]


def prologue(g):
    L_ = g.lines
    L_ += ["s_nop 4"]
    for qb in range(2):
        L_ += [f"v_mov_b32 {v(M(qb))}, 0xff800000", f"v_mov_b32 {v(L(qb))}, 0"]
    L_ += [f"v_accvgpr_write_b32 {a_(r)}, 0" for r in range(32 * DB)]
    L_ += [f"s_mov_b32 {s_(S_BIG)}, 0x53800000", f"s_mov_b32 {s_(S_I)}, 0",
           f"s_sub_u32 {s_(S_NTM1)}, {s_(S_NT)}, 1",
           # the steady iteration that masks the next tile: n-2 if the last tile is partial
           f"s_sub_u32 {s_(S_MASKAT)}, {s_(S_NT)}, 2",
           f"s_and_b32 {s_(S_TMP)}, {s_(S_KVLEN)}, 63",
           f"s_cmp_eq_u32 {s_(S_TMP)}, 0",
           f"s_cselect_b32 {s_(S_MASKAT)}, -1, {s_(S_MASKAT)}"]
    # K_0, K_1, V_0, K_2, V_1
    for desc, ring, t in ((S_KD, KRING, 0), (S_KD, KRING, 1), (S_VD, VRING, 0), (S_KD, KRING, 2), (S_VD, VRING, 1)):
        L_ += sum(dma_tile(desc, ring, t), []) + desc_advance(desc)
    # Q^T fragments: 16 bytes per lane per (query block, k-step), into v0-v63
    for qb in range(2):
        for s in range(KS):
            L_.append(f"global_load_dwordx4 {v(32 * qb + 4 * s, 4)}, {v(QPTR + 2 * qb, 2)}, off offset:{32 * s}")
    L_ += ["s_waitcnt vmcnt(0)"]
    for qb in range(2):
        for s in range(KS):
            for j in range(4):
                L_.append(f"v_accvgpr_write_b32 {a_(Q(qb, s) + j)}, {v(32 * qb + 4 * s + j)}")
    L_ += ["s_nop 2", "s_barrier"]
    # scores of tile 0, with the reads of iteration 0's first steps
    L_ += stream(qk_steps(0, 0), qk_steps(1, 1)[:LA], {}, {}, 0)
    # a single tile that is partial: mask it
    L_ += [f"s_cmp_eq_u32 {s_(S_NT)}, 1"]
    L_ += g.out_of_line("s_cbranch_scc1", [
        f"s_and_b32 {s_(S_TMP)}, {s_(S_KVLEN)}, 63",
        f"s_cmp_eq_u32 {s_(S_TMP)}, 0",
        f"s_cbranch_scc1 {g.label('Lpmaskskip')}"] + g.call_seq(g.label("Lmask0")) + [f"{g.label('Lpmaskskip')}:"])
    L_ += ["s_nop 7", "s_nop 7"]
    if g.fast:
        L_ += tile0_max()
    L_ += sm_ops(0, 0, 0, True) + sm_ops(0, 0, 1, True)
    L_ += [f"s_cmp_eq_u32 {s_(S_NT)}, 1", f"s_cbranch_scc1 {g.label('Llast0')}"]
    # the last iteration a block of four may run: n-2, or n-3 when the last
    # tile is partial (iteration n-2 masks it); the first block runs if
    # iterations 0..3 fit below it
    L_ += [f"s_sub_i32 {s_(S_LIM)}, {s_(S_NT)}, 2",
           f"s_and_b32 {s_(S_TMP)}, {s_(S_KVLEN)}, 63",
           f"s_cmp_lg_u32 {s_(S_TMP)}, 0",
           f"s_cselect_b32 {s_(S_TMP)}, 1, 0",
           f"s_sub_i32 {s_(S_LIM)}, {s_(S_LIM)}, {s_(S_TMP)}",
           f"s_cmp_ge_i32 {s_(S_LIM)}, 3",
           f"s_cbranch_scc0 {g.label('Ltail')}"]


def generate(fast=False):
    g = Gen(fast)
    prologue(g)
    # blocks of four steady iterations i..i+3 while i + 3 <= S_LIM
    g.lines += [f"{g.label('Lloop')}:"]
    for u in range(4):
        iteration(g, u, tests=False)
    g.lines += [f"s_add_u32 {s_(S_TMP)}, {s_(S_I)}, 3",
                f"s_cmp_le_i32 {s_(S_TMP)}, {s_(S_LIM)}",
                f"s_cbranch_scc1 {g.label('Lloop')}",
                f"s_cmp_eq_u32 {s_(S_I)}, {s_(S_NTM1)}",
                f"s_cbranch_scc1 {g.label('Llast0')}"]
    # the remaining steady iterations (at most four), each with the exit
    # test and the mask of a partial last tile
    g.lines += [f"{g.label('Ltail')}:"]
    for u in range(4):
        iteration(g, u)
    g.lines += [f"s_branch {g.label('Ltail')}"]
    for u in range(4):
        last_iteration(g, u)
    for par in range(2):
        if not fast:
            slow_block(g, par)
        mask_block(g, par)
    g.lines += g.cold
    g.lines += [f"{g.label('Ldone')}:", "s_waitcnt vmcnt(0) lgkmcnt(0)", "s_nop 7", "s_nop 7"]
    return g.lines


# ---------------------------------------------------------------- checks
def regs_of(tok):
    """set of ('v'|'a', index) named by an operand token"""
    tok = tok.strip().lstrip("-")
    if tok[:2] in ("v[", "a["):
        lo, hi = tok[2:-1].split(":")
        return {(tok[0], i) for i in range(int(lo), int(hi) + 1)}
    if len(tok) > 1 and tok[0] in "va" and tok[1:].isdigit():
        return {(tok[0], int(tok[1:]))}
    return set()


def operands(ln):
    op = ln.split()[0]
    return op, [t.strip().split(" ")[0] for t in ln[len(op):].split(",")]


def check_hazards(lines):
    """Straight-line check of the hand-placed distances, in issued
    instructions (s_nop n counts n+1): an MFMA result before any other use
    >= 12 (8-pass XDL write, gfx950); a VALU write before an MFMA reads it
    >= 3; a v_exp result before its use >= 2.  The state is dropped after an
    unconditional branch: code after one is reached only through a label,
    and every such block starts well clear of the MFMAs before its branch."""
    last_mfma, last_valu, last_trans = {}, {}, {}
    pos = 0
    problems = []
    for ln in lines:
        if ln.endswith(":"):
            continue
        op, ops = operands(ln)
        if op in ("s_branch", "s_setpc_b64"):
            last_mfma.clear(); last_valu.clear(); last_trans.clear()
            continue
        if op == "s_nop":
            pos += int(ln.split()[1]) + 1
            continue
        pos += 1
        dst = regs_of(ops[0]) if ops and ops[0] else set()
        srcs = set()
        for t in ops[1:]:
            srcs |= regs_of(t)
        if op.startswith("v_mfma"):
            for r in srcs:
                if r in last_valu and pos - last_valu[r] < 3:
                    problems.append(f"VALU->MFMA {r} dist {pos - last_valu[r]}: {ln}")
            c_src = regs_of(ops[3]) if len(ops) > 3 else set()
            for r in srcs - c_src:
                if r in last_mfma and pos - last_mfma[r] < 12:
                    problems.append(f"MFMA->MFMA A/B {r}: {ln}")
            for r in dst:
                last_mfma[r] = pos
        elif op.startswith(("v_", "ds_", "buffer_", "global_")):
            for r in srcs | dst:
                if r in last_mfma and pos - last_mfma[r] < 12:
                    problems.append(f"MFMA->{op} {r} dist {pos - last_mfma[r]}: {ln}")
            for r in srcs:
                if r in last_trans and pos - last_trans[r] < 2:
                    problems.append(f"trans->{op} {r}: {ln}")
            if op.startswith("v_"):
                for r in dst:
                    last_valu[r] = pos
                    if op.startswith("v_exp"):
                        last_trans[r] = pos
    return problems


def check_fragments(lines):
    """Fragment buffers: an LDS read into a buffer comes after both MFMAs of
    the buffer's previous fragment, and an MFMA reading a buffer is preceded
    by a wait that leaves no read of that buffer outstanding (LDS reads
    return in order: lgkmcnt(n) leaves the last n outstanding)."""
    problems = []
    outstanding = []              # buffers of LDS reads in issue order
    used = {}                     # buffer -> MFMAs since its last read
    for ln in lines:
        if ln.endswith(":"):
            continue
        op, ops = operands(ln)
        if op in ("s_branch", "s_setpc_b64"):
            outstanding.clear(); used.clear()
            continue
        if op.startswith("ds_read"):
            r = min(i for (_, i) in regs_of(ops[0]))
            b = (r - 192) // 4
            if "tr_b16" not in op or (r - 192) % 4 == 0:
                if used.get(b, 2) < 2:
                    problems.append(f"buffer {b} reread after {used[b]} MFMAs: {ln}")
                used[b] = 0
            outstanding.append(b)
        elif op == "s_waitcnt" and "lgkmcnt" in ln:
            n = int(ln.split("lgkmcnt(")[1].split(")")[0])
            outstanding = outstanding[len(outstanding) - n:] if n else []
        elif op.startswith("v_mfma"):
            r = min(i for (_, i) in regs_of(ops[1]))
            if 192 <= r < 224:
                b = (r - 192) // 4
                if b in outstanding:
                    problems.append(f"buffer {b} used with its read outstanding: {ln}")
                used[b] = used.get(b, 0) + 1
    return problems


def write(d):
    configure(d)
    forms = {"LOOP": generate(), "FAST": generate(fast=True)}
    for name, lines in forms.items():
        probs = check_hazards(lines) + check_fragments(lines)
        if probs:
            print("\n".join(probs[:40]))
            print(f"D={d} {name}: {len(probs)} problems")
            sys.exit(1)
    here = os.path.dirname(os.path.abspath(__file__))
    with open(os.path.join(here, f"attn_d{d}_loop.inc"), "w") as f:
        f.write("// Generated by gen_attn_loop.py from the schedule described there.\n")
        for name, lines in forms.items():
            f.write(f"// D={d} {name}: {len(lines)} lines, {sum(1 for x in lines if x.startswith('v_mfma'))} MFMAs.\n")
            f.write(f"#define DITANGO_D{d}_{name}_ASM \\\n  \"")
            f.write("\\n\\t".join(lines))
            f.write("\\n\"\n")
        # registers the block writes besides its outputs: scores,
        # probabilities, fragments, temporaries, tile sums (the Q address
        # registers v64-v67 are in/out operands), the Q^T AGPRs, scalar
        # scratch
        clob = [f'"v{i}"' for i in range(0, 64)] + [f'"v{i}"' for i in range(68, 230)]
        clob += [f'"a{i}"' for i in range(128, Q(1, KS - 1) + 4)]
        clob += [f'"s{i}"' for i in SCRATCH_SGPRS]
        clob += ['"m0"', '"vcc"', '"scc"', '"memory"']
        f.write(f"#define DITANGO_D{d}_LOOP_CLOBBERS \\\n  " + ", ".join(clob) + "\n")
    print(f"D={d}: {len(forms['LOOP'])} + {len(forms['FAST'])} lines")


def main():
    for d in (128, 64):
        write(d)


if __name__ == "__main__":
    main()
