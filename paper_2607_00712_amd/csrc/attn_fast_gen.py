"""Generates attn_fast.s: the gfx950 assembly of the head_dim-128 chunk
attention kernel (Sec. 2 Eq. 3 over the key sets of Sec. 3.4 Eq. 7-8, with the
dual-stream snapshot that gives the Eq. 11-12 fusion in one pass).

Why assembly: with 64 queries per wave and one wave per SIMD, the K and V
operands staged in LDS serve two 32-query blocks each (half the LDS operand
traffic of 32 queries per wave), and the wave must hide its own softmax work
behind its own matrix instructions. The loop is software-pipelined over
32-key halves h: phase A(h) issues the score MFMAs of half h+1 for both query
blocks while the VALU computes the softmax of half h for block 1; phase B(h)
issues the P V MFMAs of half h for both blocks while the VALU computes the
softmax of half h+1 for block 0. Every phase pairs 16 MFMAs with one block's
softmax, interleaved instruction by instruction.

Work decomposition, tile enumeration, LDS swizzles, the online softmax with a
lazy reference (exp2 with the scale folded in, the LSE from the fp32 sum of
the unrounded weights, O normalised by the sum of the bf16-rounded weights)
and the partial-result layout of the split are those of the C++ kernel in
attn_chunk.hip. Given counters, this kernel completes its split work items
itself (the split fold below); without them the merge kernel there combines
the partial results.

Run as a script it prints the assembly; build.py assembles it into a code
object that the library embeds and loads per device.
"""

import sys

KNAME = "ispa_attn_fast_d128"
ARGS_BYTES = 192

# ---------------------------------------------------------------- registers
# VGPRs
V_TID, V_LANE = 0, 1
V_KOFF = 2          # 8: K operand read addresses (buffer 0, half 0)
V_VADDR = 10        # 8: V transpose-read addresses, [h2 * 4 + db] (include the V region base)
V_STK = 18          # 4: staging voffsets of the K loads q = 0..3
V_STV = 22          # 4: staging voffsets of the V loads
V_QOFF = 26         # 2: Q load voffsets of query blocks 0 / 1
V_ST = (28, 34)     # per block: m, lr, -m c, l, lr of the current half, alpha (lr: VALU weight sums)
V_T = 40            # 16 temporaries v40..v55
V_P1 = 56           # 8: P^T of block 1 (slice 0: +0..3, slice 1: +4..7)
V_Y = 64            # 16: scores of block 0 (next half)
V_Z = (80, 96)      # 16 each: scores of block 1, by half parity
V_P0 = (112, 120)   # 8 each: P^T of block 0, by half parity
V_O = (128, 192)    # 64 each: O^T of block 0 / 1, dBlock db at +16 db
# AGPRs
A_Q = (0, 32)       # Q^T operands of block 0 / 1, slice kk at +4 kk
A_K = 64            # K operands of one half, slice kk at +4 kk
A_V = 96            # V^T operands of one half, slice s and dBlock db at +16 s + 4 db
# the normaliser of O: "mfma16", the sum of the bf16-rounded weights on the
# matrix cores, two 16x16x32 MFMAs per block and half whose A operand selects
# the lanes of one query (P^T in the 32x32x16 B layout read as a 16x16x32 B
# operand: lanes 0-15 / 32-47 hold queries 0-15, lanes 16-31 / 48-63 queries
# 16-31, so row 0 of the product sums queries 0-15 and row 1 queries 16-31);
# "mfma", the same sum with 32x32x16 MFMAs and an all-ones operand (twice the
# passes); "valu", that sum on the VALU (v_dot2c per pair); "fp32", the fp32
# sum l of the unrounded weights that the LSE uses as well. "fp32" needs no
# extra matrix instructions and runs 6.7% faster than "mfma" at the chip's
# power limit, but the sum of the rounded weights cancels their mean rounding
# error in O (the weights applied then sum to exactly 1): without it the
# error on small windows grows by 10-45%, past the 2e-2 of the output RMS
# that parity allows in one case
NORM = "mfma16"
SUMS_ON_MFMA = NORM in ("mfma", "mfma16")
N_LR = 4 if NORM == "mfma16" else 16  # accumulator registers of the sums per block
A_ONES = 128        # the bf16 A operand of the sum MFMAs (all ones, or the lane selector)
A_LR = (132, 132 + N_LR)  # the sums, per block
N_AGPR = 132 + 2 * N_LR if SUMS_ON_MFMA else 128
BF16_ONES = "0x3f803f80"
# phase schedule: spread the non-matrix instructions by estimated issue cost
BALANCED = True

# SGPRs
S_ARG = 8           # kernel arguments s[8:55]
S_RK, S_RV = 56, 60           # staging buffer resources
S_RQ = 64                     # Q resource (piece start) / scratch
S_RO, S_RL = 68, 72           # output O and LSE resources (write_state)
S_G, S_U0, S_U1, S_ITEM, S_TA, S_TB, S_T, S_FL = 76, 77, 78, 79, 80, 81, 82, 83
S_SLOT, S_HEAD, S_QTILE, S_HOFF2, S_WAVE, S_WAVE4K, S_QROWB, S_IFIRST = 84, 85, 86, 87, 88, 89, 90, 91
S_NV = 92                     # 4: valid keys of the tiles in the LDS ring
S_REC0 = 96                   # 256 - 2 ld: buffer records of a tile are nv * 2 ld + S_REC0
S_LD128 = 97                  # 128 ld: bytes of 64 rows
S_BUDGET = 98
# staging cursor: the next tile to load starts at key S_SKEY of range S_SRNG,
# which ends at key S_SEND; S_SOFF (64-bit) is the byte offset of that key's
# row slice of this head
S_SKEY, S_SEND, S_SOFF, S_SRNG = 3, 4, 5, 7
S_X, S_Y, S_W = 99, 100, 101  # scratch

# kernel-argument SGPRs (byte offset / 4 + S_ARG)
def arg(off):
    return S_ARG + off // 4

A_QPTR, A_KPTR, A_VPTR, A_OUT, A_LSE, A_OUTL, A_LSEL, A_PO, A_PL = (arg(o) for o in range(0, 72, 8))
A_U, A_LD, A_NQ, A_QT, A_T, A_LT, A_NSEG, A_MAXP, A_PERXCD, A_NLOG = (arg(o) for o in range(72, 112, 4))
A_B0, A_E0, A_B1, A_E1, A_B2, A_E2, A_TB1, A_TB2 = (arg(o) for o in range(112, 144, 4))
A_SCALE, A_C, A_LAZY, A_DUAL, A_NEGC, A_LD2, A_LD4 = (arg(o) for o in range(144, 172, 4))

A_CTR = arg(176)                # split fold: counters [item][stream][wave] (null: no fold)
# SGPRs of the split fold (argument registers that only the setup reads, and padding)
S_MFLAG = 54                    # bit w: this piece completes stream w of its item
S_GLO, S_GHI, S_GG, S_SL = 34, 35, 51, 55

K_REGION, V_REGION, BUF_BYTES, HALF_BYTES = 0, 65536, 16384, 8192
LDS_BYTES = 131072


def sp(r, n=1):
    return f"s{r}" if n == 1 else f"s[{r}:{r + n - 1}]"


def vp(r, n=1):
    return f"v{r}" if n == 1 else f"v[{r}:{r + n - 1}]"


def ap(r, n=1):
    return f"a{r}" if n == 1 else f"a[{r}:{r + n - 1}]"


class Gen:
    def __init__(self):
        self.lines = []
        self.ool = []       # out-of-line blocks (rare paths), emitted after the kernel body
        self.uid = 0

    def new_uid(self):
        self.uid += 1
        return self.uid

    def emit(self, *ins):
        for i in ins:
            self.lines.append("  " + i if not i.endswith(":") else i)

    def label(self, name):
        self.lines.append(name + ":")

    # ---------------------------------------------------------------- helpers
    def udiv(self, s_out, s_num, s_den):
        """s_out = s_num / s_den (unsigned 32-bit; s_den > 0), through the VALU."""
        t0, t1, t2, t3 = V_T, V_T + 1, V_T + 2, V_T + 3
        self.emit(f"v_cvt_f32_u32_e32 {vp(t0)}, {sp(s_den)}",
                  f"s_sub_i32 {sp(S_W)}, 0, {sp(s_den)}",
                  f"v_rcp_iflag_f32_e32 {vp(t0)}, {vp(t0)}",
                  "s_nop 0",
                  f"v_mul_f32_e32 {vp(t0)}, 0x4f7ffffe, {vp(t0)}",
                  f"v_cvt_u32_f32_e32 {vp(t0)}, {vp(t0)}",
                  f"v_mul_lo_u32 {vp(t1)}, {sp(S_W)}, {vp(t0)}",
                  f"v_mul_hi_u32 {vp(t1)}, {vp(t0)}, {vp(t1)}",
                  f"v_add_u32_e32 {vp(t0)}, {vp(t0)}, {vp(t1)}",
                  f"v_mov_b32_e32 {vp(t2)}, {sp(s_num)}",
                  f"v_mul_hi_u32 {vp(t0)}, {vp(t2)}, {vp(t0)}",
                  f"v_mul_lo_u32 {vp(t1)}, {vp(t0)}, {sp(s_den)}",
                  f"v_sub_u32_e32 {vp(t2)}, {vp(t2)}, {vp(t1)}",
                  f"v_add_u32_e32 {vp(t3)}, 1, {vp(t0)}",
                  f"v_cmp_le_u32_e32 vcc, {sp(s_den)}, {vp(t2)}",
                  f"v_subrev_u32_e32 {vp(t1)}, {sp(s_den)}, {vp(t2)}",
                  "s_nop 1",
                  f"v_cndmask_b32_e32 {vp(t0)}, {vp(t0)}, {vp(t3)}, vcc",
                  f"v_cndmask_b32_e32 {vp(t2)}, {vp(t2)}, {vp(t1)}, vcc",
                  f"v_add_u32_e32 {vp(t3)}, 1, {vp(t0)}",
                  f"v_cmp_le_u32_e32 vcc, {sp(s_den)}, {vp(t2)}",
                  "s_nop 1",
                  f"v_cndmask_b32_e32 {vp(t0)}, {vp(t0)}, {vp(t3)}, vcc",
                  "s_nop 1",
                  f"v_readfirstlane_b32 {sp(s_out)}, {vp(t0)}",
                  "s_nop 4")

    def mul64(self, s_lo, s_hi, s_a, s_b):
        """s_hi:s_lo = s_a * s_b (unsigned 32 x 32 -> 64)."""
        self.emit(f"s_mul_hi_u32 {sp(s_hi)}, {sp(s_a)}, {sp(s_b)}",
                  f"s_mul_i32 {sp(s_lo)}, {sp(s_a)}, {sp(s_b)}")

    def add64_to(self, s_dst, s_base, s_lo, s_hi):
        """s_dst:s_dst+1 = s_base:s_base+1 + s_hi:s_lo."""
        self.emit(f"s_add_u32 {sp(s_dst)}, {sp(s_base)}, {sp(s_lo)}",
                  f"s_addc_u32 {sp(s_dst + 1)}, {sp(s_base + 1)}, {sp(s_hi)}")

    # ---------------------------------------------------------------- staging
    def stage_init(self, s_tile):
        """Points the staging cursor at tile s_tile (a tile of the piece, so
        below the item's tile count): its range, first key and row offset."""
        b, e, f = S_RO, S_RO + 1, S_RO + 2   # (free outside write_state)
        self.emit(f"s_mov_b32 {sp(b)}, {sp(A_B0)}", f"s_mov_b32 {sp(e)}, {sp(A_E0)}", f"s_mov_b32 {sp(f)}, 0",
                  f"s_mov_b32 {sp(S_SRNG)}, 0",
                  f"s_cmp_ge_i32 {sp(s_tile)}, {sp(A_TB1)}",
                  f"s_cselect_b32 {sp(b)}, {sp(A_B1)}, {sp(b)}",
                  f"s_cselect_b32 {sp(e)}, {sp(A_E1)}, {sp(e)}",
                  f"s_cselect_b32 {sp(f)}, {sp(A_TB1)}, {sp(f)}",
                  f"s_cselect_b32 {sp(S_SRNG)}, 1, {sp(S_SRNG)}",
                  f"s_cmp_ge_i32 {sp(s_tile)}, {sp(A_TB2)}",
                  f"s_cselect_b32 {sp(b)}, {sp(A_B2)}, {sp(b)}",
                  f"s_cselect_b32 {sp(e)}, {sp(A_E2)}, {sp(e)}",
                  f"s_cselect_b32 {sp(f)}, {sp(A_TB2)}, {sp(f)}",
                  f"s_cselect_b32 {sp(S_SRNG)}, 2, {sp(S_SRNG)}",
                  f"s_sub_i32 {sp(f)}, {sp(s_tile)}, {sp(f)}",
                  f"s_lshl_b32 {sp(f)}, {sp(f)}, 6",
                  f"s_add_i32 {sp(S_SKEY)}, {sp(b)}, {sp(f)}",
                  f"s_mov_b32 {sp(S_SEND)}, {sp(e)}")
        self.emit(*self.cursor_offset())

    @staticmethod
    def cursor_offset():
        """S_SOFF = S_SKEY * 2 ld + 2 head_offset (64-bit)."""
        return [f"s_mul_hi_u32 {sp(S_SOFF + 1)}, {sp(S_SKEY)}, {sp(A_LD2)}",
                f"s_mul_i32 {sp(S_SOFF)}, {sp(S_SKEY)}, {sp(A_LD2)}",
                f"s_add_u32 {sp(S_SOFF)}, {sp(S_SOFF)}, {sp(S_HOFF2)}",
                f"s_addc_u32 {sp(S_SOFF + 1)}, {sp(S_SOFF + 1)}, 0"]

    def stage_list(self, s_tile, buf):
        """Direct HBM -> LDS loads of key tile s_tile (K and V, 64 rows, the
        tile under the staging cursor) into ring buffer `buf`, its valid-key
        count into s_nv[buf], and the cursor moved to the next tile, as an
        instruction list. A tile at or past the piece end (s_tile >= tb) gets
        a resource with no records: its loads fetch nothing and fill the (then
        unused) buffer with zeros, so the launch needs no branch and every
        tile step issues the same number of loads. The cursor walks the key
        ranges in order (a rare branch moves it to the next non-empty range;
        past the last one it stays put with no valid keys)."""
        nv = S_NV + buf
        f = S_RO + 2
        u = self.new_uid()
        ins = [f"s_sub_i32 {sp(nv)}, {sp(S_SEND)}, {sp(S_SKEY)}",
               f"s_min_i32 {sp(nv)}, {sp(nv)}, 64",
               f"s_add_u32 {sp(S_RK)}, {sp(A_KPTR)}, {sp(S_SOFF)}\n"
               f"  s_addc_u32 {sp(S_RK + 1)}, {sp(A_KPTR + 1)}, {sp(S_SOFF + 1)}",
               f"s_add_u32 {sp(S_RV)}, {sp(A_VPTR)}, {sp(S_SOFF)}\n"
               f"  s_addc_u32 {sp(S_RV + 1)}, {sp(A_VPTR + 1)}, {sp(S_SOFF + 1)}",
               # records: the tile's valid rows (rows past them read as zero); none past the piece
               f"s_mul_i32 {sp(f)}, {sp(nv)}, {sp(A_LD2)}",
               f"s_add_u32 {sp(f)}, {sp(f)}, {sp(S_REC0)}",
               f"s_cmp_lt_i32 {sp(s_tile)}, {sp(S_TB)}\n"
               f"  s_cselect_b32 {sp(S_RK + 2)}, {sp(f)}, 0",
               f"s_mov_b32 {sp(S_RV + 2)}, {sp(S_RK + 2)}"]
        # each wave loads 16 consecutive rows, 4 per instruction: one M0 per
        # operand, the instruction offset (applied to both the memory and the
        # LDS address; the voffsets take it back out) selects the 4 rows
        kb = K_REGION + buf * BUF_BYTES
        vb = V_REGION + buf * BUF_BYTES
        ins += [f"s_add_u32 m0, {sp(S_WAVE4K)}, {kb}\n  s_nop 0"]
        ins += [f"buffer_load_dwordx4 {vp(V_STK + q)}, {sp(S_RK, 4)}, 0 offen offset:{1024 * q} lds"
                for q in range(4)]
        ins += [f"s_add_u32 m0, {sp(S_WAVE4K)}, {vb}\n  s_nop 0"]
        ins += [f"buffer_load_dwordx4 {vp(V_STV + q)}, {sp(S_RV, 4)}, 0 offen offset:{1024 * q} lds"
                for q in range(4)]
        ins += [f"s_add_u32 {sp(S_SKEY)}, {sp(S_SKEY)}, 64",
                f"s_add_u32 {sp(S_SOFF)}, {sp(S_SOFF)}, {sp(S_LD128)}\n"
                f"  s_addc_u32 {sp(S_SOFF + 1)}, {sp(S_SOFF + 1)}, 0",
                f"s_cmp_ge_i32 {sp(S_SKEY)}, {sp(S_SEND)}\n  s_cbranch_scc1 .Lnr{u}\n.Lnrback{u}:"]
        self.ool.append([f".Lnr{u}:",
                         f"s_add_u32 {sp(S_SRNG)}, {sp(S_SRNG)}, 1",
                         f"s_cmp_eq_u32 {sp(S_SRNG)}, 1",
                         f"s_cselect_b32 {sp(S_SKEY)}, {sp(A_B1)}, {sp(S_SKEY)}",
                         f"s_cselect_b32 {sp(S_SEND)}, {sp(A_E1)}, {sp(S_SEND)}",
                         f"s_cmp_eq_u32 {sp(S_SRNG)}, 2",
                         f"s_cselect_b32 {sp(S_SKEY)}, {sp(A_B2)}, {sp(S_SKEY)}",
                         f"s_cselect_b32 {sp(S_SEND)}, {sp(A_E2)}, {sp(S_SEND)}",
                         f"s_cmp_lt_u32 {sp(S_SRNG)}, 3",
                         f"s_cselect_b32 {sp(S_SEND)}, {sp(S_SEND)}, {sp(S_SKEY)}",
                         f"s_cbranch_scc0 .Lnrback{u}",
                         f"s_cmp_ge_i32 {sp(S_SKEY)}, {sp(S_SEND)}",
                         f"s_cbranch_scc1 .Lnr{u}"]
                        + self.cursor_offset()
                        + [f"s_branch .Lnrback{u}"])
        return ins

    def stage(self, s_tile, buf):
        for i in self.stage_list(s_tile, buf):
            self.emit(i)

    # ---------------------------------------------------------------- softmax
    @staticmethod
    def weights(S, nmc, P, dot=None):
        """Weights p = 2^(s c - m c) of the 16 scores S into the temporaries
        (exponentials in groups of four, each four instructions after its
        argument), the bf16 pairs into P, and the fp32 sum of the 16 unrounded
        weights into the first temporary (by pairs, then a tree)."""
        T = [V_T + i for i in range(16)]
        ins = []
        pend = []
        for g in range(4):
            idx = [4 * g + i for i in range(4)]
            ins += [f"v_fma_f32 {vp(T[i])}, {vp(S[i])}, {sp(A_C)}, {vp(nmc)}" for i in idx]
            ins += pend[:4]
            ins += [f"v_exp_f32_e32 {vp(T[i])}, {vp(T[i])}" for i in idx]
            ins += pend[4:]
            pend = []
            for pp in (2 * g, 2 * g + 1):
                a_, b_ = T[2 * pp], T[2 * pp + 1]
                pend += [f"v_cvt_pk_bf16_f32 {vp(P[pp])}, {vp(a_)}, {vp(b_)}",
                         f"v_add_f32_e32 {vp(a_)}, {vp(a_)}, {vp(b_)}"]
                if dot is not None and pp > 0:
                    pend += [f"v_dot2c_f32_bf16_e32 {vp(dot)}, {BF16_ONES}, {vp(P[pp - 1])}"]
        if dot is not None:
            ins = [f"v_mov_b32_e32 {vp(dot)}, 0"] + ins
        ins += ["s_nop 0"] + pend
        if dot is not None:
            ins += [f"v_dot2c_f32_bf16_e32 {vp(dot)}, {BF16_ONES}, {vp(P[7])}"]
        ins += [f"v_add_f32_e32 {vp(T[0])}, {vp(T[0])}, {vp(T[2])}",
                f"v_add_f32_e32 {vp(T[4])}, {vp(T[4])}, {vp(T[6])}",
                f"v_add_f32_e32 {vp(T[8])}, {vp(T[8])}, {vp(T[10])}",
                f"v_add_f32_e32 {vp(T[12])}, {vp(T[12])}, {vp(T[14])}",
                f"v_add_f32_e32 {vp(T[0])}, {vp(T[0])}, {vp(T[4])}",
                f"v_add_f32_e32 {vp(T[8])}, {vp(T[8])}, {vp(T[12])}",
                f"v_add_f32_e32 {vp(T[0])}, {vp(T[0])}, {vp(T[8])}"]
        return ins

    def softmax(self, qb, s_base, p_base, nv_reg, half):
        """The online-softmax step of query block qb over one 32-key half
        whose scores are in v[s_base:+15]: the bf16 weights into
        v[p_base:+7] and the fp32 sum of this lane's 16 weights into the first
        temporary. Returns (body, check): the body is interleaved with matrix
        instructions, the check (the trigger compare into VCC) ends the phase,
        and resolve() takes the branch and adds the sum to l.

        The reference m moves lazily: the weights are computed against the
        current m, and only when some lane's 16 weights sum to more than 2^8
        (or to inf / NaN: the first half of a piece starts from m = -inf with
        -m c = +inf) does a rare path raise m to the row maximum, recompute
        the weights and rescale l, O and the bf16 weight sums by
        alpha = 2^((m_old - m_new) c). Every weight therefore stays at or
        below 2^8, as with an explicit maximum test, without the maximum on
        the common path. The branch is taken after the phase's P V matrix
        instructions (those still apply weights of the old reference) have
        been issued; the rare path waits for them before it rescales O."""
        m, nmc, l, alpha = V_ST[qb], V_ST[qb] + 2, V_ST[qb] + 3, V_ST[qb] + 5
        lr, dot = V_ST[qb] + 1, (V_ST[qb] + 4 if NORM == "valu" else None)
        u = self.new_uid()
        T = V_T
        S = [s_base + r for r in range(16)]
        P = [p_base + i for i in range(8)]
        ins = []
        # keys past the end of a range (only in the last tile of each range)
        # (a rare-path branch and the label it returns to stay adjacent: the
        # interleaver must not move matrix or LDS instructions between them)
        ins += [f"s_cmp_lt_u32 {sp(nv_reg)}, {32 * (half + 1)}\n  s_cbranch_scc1 .Lmask{u}\n.Lmback{u}:"]
        mask = [f".Lmask{u}:",
                f"s_sub_i32 {sp(S_W)}, {sp(nv_reg)}, {32 * half}",
                f"v_lshrrev_b32_e32 {vp(T)}, 5, {vp(V_LANE)}",
                f"v_lshlrev_b32_e32 {vp(T)}, 2, {vp(T)}",
                f"v_sub_u32_e32 {vp(T)}, {sp(S_W)}, {vp(T)}",        # lim = nv - 32 half - 4 hh
                f"v_mov_b32_e32 {vp(T + 1)}, 0xff800000"]
        for r in range(16):
            c = 8 * (r >> 2) + (r & 3)    # key of register r within the half, less 4 hh
            mask += [f"v_cmp_ge_i32_e32 vcc, {c}, {vp(T)}", "s_nop 1",
                     f"v_cndmask_b32_e32 {vp(S[r])}, {vp(S[r])}, {vp(T + 1)}, vcc"]
        mask += [f"s_branch .Lmback{u}"]
        self.ool.append(mask)
        ins += self.weights(S, nmc, P, dot)
        # trigger: !(2^8 >= lane sum), true for a sum above 2^8, inf or NaN
        return ins, [f"v_cmp_nge_f32_e32 vcc, 0x43800000, {vp(T)}"]

    def resolve(self, qb, s_base, p_base):
        """The branch on a softmax step's trigger (in VCC) and the addition of
        its weight sums to l: placed after the first matrix instruction of the
        next phase (so the compare has completed when the branch reads VCC),
        before anything there overwrites the temporaries or, for block 0, the
        scores. The rare path (emitted out of line): the row maximum over the
        16 scores (a tree of depth three) and the lane pair, the new
        reference, the weights again, and the rescale of l, O and the weight
        sums."""
        m, nmc, l, alpha = V_ST[qb], V_ST[qb] + 2, V_ST[qb] + 3, V_ST[qb] + 5
        lr, dot = V_ST[qb] + 1, (V_ST[qb] + 4 if NORM == "valu" else None)
        u = self.new_uid()
        T = V_T
        S = [s_base + r for r in range(16)]
        P = [p_base + i for i in range(8)]
        out = [f"s_cbranch_vccnz .Lresc{u}\n.Lrback{u}:",
               f"v_add_f32_e32 {vp(l)}, {vp(l)}, {vp(T)}"]
        if dot is not None:
            out += [f"v_add_f32_e32 {vp(lr)}, {vp(lr)}, {vp(dot)}"]
        resc = [f".Lresc{u}:",
                f"v_maximum3_f32 {vp(T)}, {vp(S[0])}, {vp(S[1])}, {vp(S[2])}",
                f"v_maximum3_f32 {vp(T + 1)}, {vp(S[3])}, {vp(S[4])}, {vp(S[5])}",
                f"v_maximum3_f32 {vp(T + 2)}, {vp(S[6])}, {vp(S[7])}, {vp(S[8])}",
                f"v_maximum3_f32 {vp(T + 3)}, {vp(S[9])}, {vp(S[10])}, {vp(S[11])}",
                f"v_maximum3_f32 {vp(T + 4)}, {vp(S[12])}, {vp(S[13])}, {vp(S[14])}",
                f"v_maximum3_f32 {vp(T)}, {vp(T)}, {vp(T + 1)}, {vp(T + 2)}",
                f"v_maximum3_f32 {vp(T + 3)}, {vp(T + 3)}, {vp(T + 4)}, {vp(S[15])}",
                f"v_maximum3_f32 {vp(T)}, {vp(T)}, {vp(T + 3)}, {vp(T + 3)}",
                f"v_mov_b32_e32 {vp(T + 1)}, {vp(T)}",
                "s_nop 1",
                f"v_permlane32_swap_b32 {vp(T)}, {vp(T + 1)}",
                "s_nop 1",
                f"v_maximum3_f32 {vp(T + 1)}, {vp(m)}, {vp(T)}, {vp(T + 1)}",    # m_new
                f"v_sub_f32_e32 {vp(T + 2)}, {vp(m)}, {vp(T + 1)}",
                f"v_mul_f32_e32 {vp(T + 2)}, {sp(A_C)}, {vp(T + 2)}",
                f"v_exp_f32_e32 {vp(alpha)}, {vp(T + 2)}",
                f"v_mov_b32_e32 {vp(m)}, {vp(T + 1)}",
                f"v_mul_f32_e32 {vp(nmc)}, {sp(A_NEGC)}, {vp(T + 1)}",
                "s_nop 0",
                f"v_mul_f32_e32 {vp(l)}, {vp(alpha)}, {vp(l)}"]
        resc += self.weights(S, nmc, P, dot)
        # the P V instructions issued so far (old reference) have completed
        resc += ["s_nop 7", "s_nop 7", "s_nop 7"]
        resc += [f"v_mul_f32_e32 {vp(V_O[qb] + i)}, {vp(alpha)}, {vp(V_O[qb] + i)}" for i in range(64)]
        if NORM == "mfma16":
            # register 0 of lane n (< 16) sums query n, register 1 query n + 16,
            # whose alpha lane n + 16 holds; the other lanes and registers are 0
            t, a16, adr = V_T + 8, V_T + 9, V_T + 10
            resc += [f"v_add_u32_e32 {vp(adr)}, 16, {vp(V_LANE)}",
                     f"v_and_b32_e32 {vp(adr)}, 63, {vp(adr)}",
                     f"v_lshlrev_b32_e32 {vp(adr)}, 2, {vp(adr)}",
                     f"ds_bpermute_b32 {vp(a16)}, {vp(adr)}, {vp(alpha)}",
                     f"v_accvgpr_read_b32 {vp(t)}, {ap(A_LR[qb])}",
                     f"v_mul_f32_e32 {vp(t)}, {vp(alpha)}, {vp(t)}",
                     f"v_accvgpr_write_b32 {ap(A_LR[qb])}, {vp(t)}",
                     "s_waitcnt lgkmcnt(0)",
                     f"v_accvgpr_read_b32 {vp(t)}, {ap(A_LR[qb] + 1)}",
                     f"v_mul_f32_e32 {vp(t)}, {vp(a16)}, {vp(t)}",
                     f"v_accvgpr_write_b32 {ap(A_LR[qb] + 1)}, {vp(t)}"]
        elif SUMS_ON_MFMA:
            for i in range(16):
                t = V_T + 8 + (i & 7)
                resc += [f"v_accvgpr_read_b32 {vp(t)}, {ap(A_LR[qb] + i)}",
                         f"v_mul_f32_e32 {vp(t)}, {vp(alpha)}, {vp(t)}",
                         f"v_accvgpr_write_b32 {ap(A_LR[qb] + i)}, {vp(t)}"]
        elif NORM == "valu":
            resc += [f"v_mul_f32_e32 {vp(lr)}, {vp(alpha)}, {vp(lr)}"]
        resc += [f"s_branch .Lrback{u}"]
        self.ool.append(resc)
        return out

    # ---------------------------------------------------------------- matrix work
    @staticmethod
    def mfma_scores(y_reg, z_reg):
        """S^T = K Q^T of both blocks for the half whose K operands are in A_K."""
        # the two blocks' accumulation chains alternate, so that consecutive
        # MFMAs are independent
        out = []
        for kk in range(8):
            for qb, dst in ((1, z_reg), (0, y_reg)):
                c = "0" if kk == 0 else vp(dst, 16)
                out.append(f"v_mfma_f32_32x32x16_bf16 {vp(dst, 16)}, {ap(A_K + 4 * kk, 4)}, "
                           f"{ap(A_Q[qb] + 4 * kk, 4)}, {c}")
        return out

    @staticmethod
    def mfma_pv(p0_reg):
        """O^T += V^T P^T of both blocks for the half whose V operands are in A_V."""
        out = []
        for qb, p in ((0, p0_reg), (1, V_P1)):
            for s in range(2):
                for db in range(4):
                    o = vp(V_O[qb] + 16 * db, 16)
                    out.append(f"v_mfma_f32_32x32x16_bf16 {o}, {ap(A_V + 16 * s + 4 * db, 4)}, "
                               f"{vp(p + 4 * s, 4)}, {o}")
            for s in range(2 if SUMS_ON_MFMA else 0):
                acc = ap(A_LR[qb], N_LR)
                shape = "16x16x32" if NORM == "mfma16" else "32x32x16"
                out.append(f"v_mfma_f32_{shape}_bf16 {acc}, {ap(A_ONES, 4)}, {vp(p + 4 * s, 4)}, {acc}")
        return out

    @staticmethod
    def lds_k(buf, half):
        base = K_REGION + buf * BUF_BYTES + half * HALF_BYTES
        return [f"ds_read_b128 {ap(A_K + 4 * kk, 4)}, {vp(V_KOFF + kk)} offset:{base}" for kk in range(8)]

    @staticmethod
    def lds_v(buf, half):
        out = []
        for s in range(2):
            imm = buf * BUF_BYTES + 16 * (2 * half + s) * 256
            for db in range(4):
                a = A_V + 16 * s + 4 * db
                out.append(f"ds_read_b64_tr_b16 {ap(a, 2)}, {vp(V_VADDR + db)} offset:{imm}")
                out.append(f"ds_read_b64_tr_b16 {ap(a + 2, 2)}, {vp(V_VADDR + 4 + db)} offset:{imm}")
        return out

    @staticmethod
    def cost(item):
        """Issue cycles of an instruction-list item for one wave (estimates:
        a VALU op about 4, a transcendental 8, an LDS or buffer op 4 / 8)."""
        c = 0
        for ln in item.split("\n"):
            t = ln.strip()
            if not t or t.endswith(":"):
                continue
            op = t.split()[0]
            if op.startswith(("v_exp", "v_log", "v_rcp")):
                c += 8
            elif op.startswith("v_"):
                c += 4
            elif op.startswith("ds_"):
                c += 4
            elif op.startswith("buffer_"):
                c += 8
            elif op == "s_nop":
                c += int(t.split()[1]) + 1
            else:
                c += 1
        return c

    def phase(self, mfma, lds, valu, tail=(), lds_start=2, stage=(), pre=()):
        """Interleave 16 or 20 (or 0) MFMAs with LDS reads, the staging list
        and a VALU list, then the tail. The LDS reads go two per matrix
        instruction from the third one on (the operands they overwrite may
        still be read by the previous phase's last matrix instructions); the
        staging and VALU lists are merged in proportion to their issue cost
        and spread so that every matrix instruction carries about the same
        issue time, with at most one buffer load after each."""
        self.emit("s_waitcnt lgkmcnt(0)")
        if not mfma:
            for i in list(pre) + list(lds) + list(stage) + list(valu) + list(tail):
                self.emit(i)
            return
        n = len(mfma)
        lds_slots = [[] for _ in range(n)]
        if lds:
            span = max(1, min(n - lds_start, 8))
            per = -(-len(lds) // span)
            for k, i in enumerate(lds):
                lds_slots[lds_start + k // per].append(i)
        if not BALANCED:
            valu = list(stage) + list(valu)
            per_v = -(-len(valu) // n)
            for s_ in range(n):
                self.emit(mfma[s_], *(pre if s_ == 0 else ()), *lds_slots[s_], *valu[s_ * per_v:(s_ + 1) * per_v])
            for i in list(valu[n * per_v:]) + list(tail):
                self.emit(i)
            return
        # merge the staging and VALU lists by cost (their orders are kept)
        cs, cv = sum(map(self.cost, stage)), sum(map(self.cost, valu))
        merged, a, b, da, db = [], 0, 0, 0, 0
        while a < len(stage) or b < len(valu):
            if b >= len(valu) or (a < len(stage) and da * max(cv, 1) <= db * max(cs, 1)):
                merged.append(stage[a]); da += self.cost(stage[a]); a += 1
            else:
                merged.append(valu[b]); db += self.cost(valu[b]); b += 1
        total = sum(map(self.cost, merged)) + sum(self.cost(i) for sl in lds_slots for i in sl)
        k, done, cum_lds = 0, 0, 0
        for s_ in range(n):
            self.emit(mfma[s_])
            if s_ == 0:
                for i in pre:
                    self.emit(i)
            for i in lds_slots[s_]:
                self.emit(i)
                cum_lds += self.cost(i)
            target = total * (s_ + 1) / n - cum_lds
            vm = 0
            while k < len(merged) and (done < target or s_ == n - 1):
                it = merged[k]
                if "buffer_load" in it:
                    if vm:
                        break
                    vm = 1
                self.emit(it)
                done += self.cost(it)
                k += 1
        for i in list(merged[k:]) + list(tail):
            self.emit(i)

    # ---------------------------------------------------------------- output
    @staticmethod
    def lr16(qb, dst, t1, t2):
        """dst = the sum of the bf16-rounded weights of this lane's query
        (lane & 31) from the 16x16 sum accumulator of block qb: register 0 of
        lane q for q < 16, register 1 of lane q - 16 otherwise (the sum MFMAs
        have completed)."""
        return [f"v_accvgpr_read_b32 {vp(dst)}, {ap(A_LR[qb])}",
                f"v_accvgpr_read_b32 {vp(t1)}, {ap(A_LR[qb] + 1)}",
                f"v_and_b32_e32 {vp(t2)}, 15, {vp(V_LANE)}",
                f"v_lshlrev_b32_e32 {vp(t2)}, 2, {vp(t2)}",
                f"ds_bpermute_b32 {vp(dst)}, {vp(t2)}, {vp(dst)}",
                f"ds_bpermute_b32 {vp(t1)}, {vp(t2)}, {vp(t1)}",
                f"v_and_b32_e32 {vp(t2)}, 16, {vp(V_LANE)}",
                f"v_cmp_ne_u32_e32 vcc, 0, {vp(t2)}",
                "s_waitcnt lgkmcnt(0)",
                f"v_cndmask_b32_e32 {vp(dst)}, {vp(dst)}, {vp(t1)}, vcc"]

    def write_state(self, rows, which):
        """Normalised O and LSE of both blocks. rows: to the output rows
        (out / lse, or out_local / lse_local when which = 1); else to partial
        slot S_SLOT (part `which`)."""
        u = self.new_uid()
        T = V_T
        # partial results are stored coherent at device scope (sc1), so that a
        # piece on another XCD reads them (also sc1) once the count says so
        coh = "" if rows else " sc1"
        if rows:
            self.row_resources(which)
        else:
            # O: part_o + ((slot * 2 + which) * 256 + wave * 64) * 512
            self.emit(f"s_lshl_b32 {sp(S_Y)}, {sp(S_SLOT)}, 1")
            if which:
                self.emit(f"s_add_u32 {sp(S_Y)}, {sp(S_Y)}, 1")
            self.emit(f"s_lshl_b32 {sp(S_Y)}, {sp(S_Y)}, 8",
                      f"s_lshl_b32 {sp(S_W)}, {sp(S_WAVE)}, 6",
                      f"s_add_u32 {sp(S_Y)}, {sp(S_Y)}, {sp(S_W)}",           # first query of this wave's rows
                      f"s_mov_b32 {sp(S_RO + 2)}, 512")
            self.mul64(S_X, S_W, S_Y, S_RO + 2)
            self.add64_to(S_RO, A_PO, S_X, S_W)
            self.emit(f"s_mov_b32 {sp(S_RO + 2)}, 32768", f"s_mov_b32 {sp(S_RO + 3)}, 0x20000")
            self.emit(f"s_mov_b32 {sp(S_RL + 2)}, 4")
            self.mul64(S_X, S_W, S_Y, S_RL + 2)
            self.add64_to(S_RL, A_PL, S_X, S_W)
            self.emit(f"s_mov_b32 {sp(S_RL + 2)}, 256", f"s_mov_b32 {sp(S_RL + 3)}, 0x20000",
                      f"s_mov_b32 {sp(S_X)}, 512")
        # every P V MFMA has completed (the O registers are read below)
        self.emit("s_nop 7", "s_nop 7", "s_nop 7",
                  f"v_and_b32_e32 {vp(T)}, 31, {vp(V_LANE)}",              # ql
                  f"v_lshrrev_b32_e32 {vp(T + 1)}, 5, {vp(V_LANE)}",
                  f"v_lshlrev_b32_e32 {vp(T + 1)}, 4, {vp(T + 1)}",         # 16 hh
                  f"v_mov_b32_e32 {vp(V_Y)}, 0x40000000")                   # an offset past every record (the scores are dead here)
        for qb in range(2):
            m, l = V_ST[qb], V_ST[qb] + 3
            if NORM == "mfma":
                self.emit(f"v_accvgpr_read_b32 {vp(T + 4)}, {ap(A_LR[qb])}")      # lr total
            elif NORM == "mfma16":
                self.emit(*self.lr16(qb, T + 4, T + 5, T + 6))                     # lr total
            elif NORM == "valu":
                self.emit(f"v_mov_b32_e32 {vp(T + 4)}, {vp(V_ST[qb] + 1)}", f"v_mov_b32_e32 {vp(T + 5)}, {vp(V_ST[qb] + 1)}",
                          "s_nop 1",
                          f"v_permlane32_swap_b32 {vp(T + 4)}, {vp(T + 5)}",
                          "s_nop 1",
                          f"v_add_f32_e32 {vp(T + 4)}, {vp(T + 4)}, {vp(T + 5)}")  # lr total
            self.emit(f"v_mov_b32_e32 {vp(T + 2)}, {vp(l)}", f"v_mov_b32_e32 {vp(T + 3)}, {vp(l)}",
                      "s_nop 1",
                      f"v_permlane32_swap_b32 {vp(T + 2)}, {vp(T + 3)}",
                      "s_nop 1",
                      f"v_add_f32_e32 {vp(T + 2)}, {vp(T + 2)}, {vp(T + 3)}")   # l total
            if NORM == "fp32":
                self.emit(f"v_mov_b32_e32 {vp(T + 4)}, {vp(T + 2)}")
            self.emit(f"v_rcp_f32_e32 {vp(T + 4)}, {vp(T + 4)}",
                      f"v_add_u32_e32 {vp(T + 6)}, {32 * qb}, {vp(T)}",
                      f"v_mul_lo_u32 {vp(T + 7)}, {vp(T + 6)}, {sp(S_X)}",
                      f"v_add_u32_e32 {vp(T + 7)}, {vp(T + 7)}, {vp(T + 1)}")  # O voffset
            for db in range(4):
                for j in range(4):
                    d = T + 8 + 4 * (j & 1)
                    src = V_O[qb] + 16 * db + 4 * j
                    for i in range(4):
                        self.emit(f"v_mul_f32_e32 {vp(d + i)}, {vp(T + 4)}, {vp(src + i)}")
                    self.emit(f"buffer_store_dwordx4 {vp(d, 4)}, {vp(T + 7)}, {sp(S_RO, 4)}, 0 offen "
                              f"offset:{128 * db + 32 * j}{coh}")
            # LSE = m scale + ln(l total), from the lanes of the lower half
            self.emit(f"v_log_f32_e32 {vp(T + 2)}, {vp(T + 2)}",
                      f"v_lshlrev_b32_e32 {vp(T + 6)}, 2, {vp(T + 6)}",
                      f"v_cmp_ne_u32_e32 vcc, 0, {vp(T + 1)}",
                      f"v_mul_f32_e32 {vp(T + 2)}, 0x3f317218, {vp(T + 2)}",
                      f"v_fma_f32 {vp(T + 3)}, {vp(m)}, {sp(A_SCALE)}, {vp(T + 2)}",
                      f"v_cndmask_b32_e32 {vp(T + 6)}, {vp(T + 6)}, {vp(V_Y)}, vcc",
                      "s_nop 1",
                      f"buffer_store_dword {vp(T + 3)}, {vp(T + 6)}, {sp(S_RL, 4)}, 0 offen{coh}")
        self.emit("s_waitcnt vmcnt(0)")
        del u

    def row_resources(self, which):
        """S_RO, S_RL: this wave's rows of the output O and LSE of stream
        `which` (rows past n_q have no records; no LSE records when its
        pointer is null); S_X = the lane stride of O (bytes per row)."""
        optr, lptr = (A_OUT, A_LSE) if which == 0 else (A_OUTL, A_LSEL)
        # O: base = out + (qrow_b * ld + hoff) * 4; this wave's rows that exist
        self.mul64(S_X, S_Y, S_QROWB, A_LD4)
        self.emit(f"s_lshl_b32 {sp(S_W)}, {sp(S_HOFF2)}, 1",
                  f"s_add_u32 {sp(S_X)}, {sp(S_X)}, {sp(S_W)}", f"s_addc_u32 {sp(S_Y)}, {sp(S_Y)}, 0")
        self.add64_to(S_RO, optr, S_X, S_Y)
        self.emit(f"s_sub_i32 {sp(S_W)}, {sp(A_NQ)}, {sp(S_QROWB)}",
                  f"s_min_i32 {sp(S_W)}, {sp(S_W)}, 64",
                  f"s_max_i32 {sp(S_W)}, {sp(S_W)}, 0",
                  f"s_mul_i32 {sp(S_RO + 2)}, {sp(S_W)}, {sp(A_LD4)}",     # (covers the rows' head slices)
                  f"s_mov_b32 {sp(S_RO + 3)}, 0x20000",
                  f"s_mov_b32 {sp(S_X)}, {sp(A_LD4)}")                    # lane stride
        # LSE: base = lse + (head * n_q + qrow_b) * 4; none when the pointer is null
        self.emit(f"s_mul_i32 {sp(S_Y)}, {sp(S_HEAD)}, {sp(A_NQ)}",
                  f"s_add_u32 {sp(S_Y)}, {sp(S_Y)}, {sp(S_QROWB)}",
                  f"s_mul_hi_u32 {sp(S_RL + 3)}, {sp(S_Y)}, 4",
                  f"s_mul_i32 {sp(S_Y)}, {sp(S_Y)}, 4")
        self.emit(f"s_add_u32 {sp(S_RL)}, {sp(lptr)}, {sp(S_Y)}",
                  f"s_addc_u32 {sp(S_RL + 1)}, {sp(lptr + 1)}, {sp(S_RL + 3)}",
                  f"s_lshl_b32 {sp(S_RL + 2)}, {sp(S_W)}, 2",
                  f"s_cmp_eq_u64 {sp(lptr, 2)}, 0",
                  f"s_cselect_b32 {sp(S_RL + 2)}, 0, {sp(S_RL + 2)}",
                  f"s_mov_b32 {sp(S_RL + 3)}, 0x20000")

    # ---------------------------------------------------------------- split fold
    # With a counter array (A_CTR non-null), the pieces of a split work item
    # complete it themselves instead of a merge kernel after the launch: every
    # piece writes its normalised partial result and LSE to its slot (as for
    # the merge kernel) with device-coherent stores, and once they are complete
    # counts itself on the item's counter of that stream with an atomic add;
    # the piece that brings the count to the number of pieces reads every
    # piece's partial back with device-coherent loads and combines them with
    # Eq. 11-12 in piece order, so the result does not depend on which piece
    # finishes last. No piece ever waits for another, and no cache is written
    # back or invalidated as a whole.
    def seg_of(self, s_out, s_unit):
        """s_out = the segment (workgroup run) that holds unit s_unit:
        ((u + 1) n_seg - 1) / units (32-bit, as the host checks)."""
        self.emit(f"s_add_u32 {sp(S_W)}, {sp(s_unit)}, 1",
                  f"s_mul_i32 {sp(S_W)}, {sp(S_W)}, {sp(A_NSEG)}",
                  f"s_sub_u32 {sp(S_Y)}, {sp(S_W)}, 1")
        self.udiv(s_out, S_Y, A_U)

    def piece_segments(self, which):
        """S_GLO, S_GHI: the first and last segments of this item's stream
        `which` (all T tiles, or the LT tiles of the local set)."""
        self.emit(f"s_mul_i32 {sp(S_GG)}, {sp(S_ITEM)}, {sp(A_T)}")
        self.seg_of(S_GLO, S_GG)
        self.emit(f"s_add_u32 {sp(S_GG)}, {sp(S_GG)}, {sp(A_T if which == 0 else A_LT)}",
                  f"s_sub_u32 {sp(S_GG)}, {sp(S_GG)}, 1")
        self.seg_of(S_GHI, S_GG)

    def counter(self, which):
        """S_RQ: the record of this wave's counter of stream `which`
        ((item * 2 + which) * 4 + wave); V_T: lane 0's offset in it, the other
        lanes' offsets past the record (so one lane accesses it)."""
        T = V_T
        self.emit(f"s_lshl_b32 {sp(S_W)}, {sp(S_ITEM)}, 5",
                  f"s_lshl_b32 {sp(S_Y)}, {sp(S_WAVE)}, 2",
                  f"s_add_u32 {sp(S_W)}, {sp(S_W)}, {sp(S_Y)}",
                  f"s_add_u32 {sp(S_RQ)}, {sp(A_CTR)}, {sp(S_W)}",
                  f"s_addc_u32 {sp(S_RQ + 1)}, {sp(A_CTR + 1)}, 0",
                  f"s_mov_b32 {sp(S_RQ + 2)}, {16 * which + 4}",
                  f"s_mov_b32 {sp(S_RQ + 3)}, 0x20000",
                  f"v_cmp_eq_u32_e32 vcc, 0, {vp(V_LANE)}",
                  f"v_mov_b32_e32 {vp(T)}, 0x40000000",
                  "s_nop 1",
                  f"v_cndmask_b32_e64 {vp(T)}, {vp(T)}, {16 * which}, vcc",
                  "s_nop 1")

    def count(self, which, done):
        """Adds this piece to its counter of stream `which` (its partial's
        device-coherent stores are complete: vmcnt(0) at the end of
        write_state); branches to `done` unless it completes the stream.
        Needs S_GLO, S_GHI."""
        T = V_T
        self.counter(which)
        self.emit(f"v_mov_b32_e32 {vp(T + 1)}, 1",
                  f"buffer_atomic_add {vp(T + 1)}, {vp(T)}, {sp(S_RQ, 4)}, 0 offen sc0",
                  "s_waitcnt vmcnt(0)",
                  f"v_readfirstlane_b32 {sp(S_Y)}, {vp(T + 1)}",
                  "s_nop 4",
                  f"s_sub_u32 {sp(S_W)}, {sp(S_GHI)}, {sp(S_GLO)}",         # pieces - 1
                  f"s_cmp_eq_u32 {sp(S_Y)}, {sp(S_W)}",
                  f"s_cbranch_scc0 {done}")

    def publish(self, which):
        """At the local snapshot inside a piece, after this piece's partial of
        stream `which` is in its slot: the count, and the merge flag (the
        merge from the slots follows at the piece end) when this piece
        completes the item's stream."""
        u = self.new_uid()
        self.emit(f"s_cmp_eq_u64 {sp(A_CTR, 2)}, 0", f"s_cbranch_scc1 .Lpub_done{u}")
        self.piece_segments(which)
        self.count(which, f".Lpub_done{u}")
        self.emit(f"s_or_b32 {sp(S_MFLAG)}, {sp(S_MFLAG)}, {1 << which}",
                  f".Lpub_done{u}:")

    def finish_stream(self, which):
        """At the end of a piece that holds part of stream `which` of its item:
        the partial to the slot and the count; the piece that completes the
        stream merges. With two pieces the merge takes this piece's own part
        from its registers, and a piece that finds the other one already
        counted merges without storing its own part."""
        u = self.new_uid()
        T = V_T
        done = f".Lfin_done{u}"
        self.emit(f"s_cmp_eq_u64 {sp(A_CTR, 2)}, 0", f"s_cbranch_scc0 .Lfin_fold{u}")
        self.write_state(False, which)
        self.emit(f"s_branch {done}", f".Lfin_fold{u}:")
        self.piece_segments(which)
        self.emit(f"s_sub_u32 {sp(S_W)}, {sp(S_GHI)}, {sp(S_GLO)}",
                  f"s_cmp_eq_u32 {sp(S_W)}, 1",
                  f"s_cbranch_scc0 .Lfin_store{u}")
        # two pieces: has the other one counted already?
        self.counter(which)
        self.emit(f"buffer_load_dword {vp(T + 1)}, {vp(T)}, {sp(S_RQ, 4)}, 0 offen sc1",
                  "s_waitcnt vmcnt(0)",
                  f"v_readfirstlane_b32 {sp(S_Y)}, {vp(T + 1)}",
                  "s_nop 4",
                  f"s_cmp_eq_u32 {sp(S_Y)}, 1",
                  f"s_cbranch_scc1 .Lfin_merge2{u}",
                  f".Lfin_store{u}:")
        self.write_state(False, which)
        self.count(which, done)
        self.emit(f"s_sub_u32 {sp(S_W)}, {sp(S_GHI)}, {sp(S_GLO)}",
                  f"s_cmp_eq_u32 {sp(S_W)}, 1",
                  f"s_cbranch_scc1 .Lfin_merge2{u}",
                  f"s_or_b32 {sp(S_MFLAG)}, {sp(S_MFLAG)}, {1 << which}",
                  f"s_branch {done}",
                  f".Lfin_merge2{u}:")
        self.merge2(which)
        self.label(done)

    def slot_resources(self, s_g, which):
        """S_RO, S_RL: this wave's rows of the partial O and LSE of stream
        `which` that segment s_g left for this item."""
        # slot of segment g: g max_pieces + item - (its first item)
        self.emit(f"s_mul_i32 {sp(S_Y)}, {sp(s_g)}, {sp(A_U)}")
        self.udiv(S_SL, S_Y, A_NSEG)
        self.udiv(S_SL, S_SL, A_T)
        self.emit(f"s_mul_i32 {sp(S_W)}, {sp(s_g)}, {sp(A_MAXP)}",
                  f"s_add_u32 {sp(S_W)}, {sp(S_W)}, {sp(S_ITEM)}",
                  f"s_sub_u32 {sp(S_SL)}, {sp(S_W)}, {sp(S_SL)}",
                  # rows of this wave in part (slot, which): ((slot * 2 + which) * 256 + 64 wave)
                  f"s_lshl_b32 {sp(S_W)}, {sp(S_SL)}, 1")
        if which:
            self.emit(f"s_add_u32 {sp(S_W)}, {sp(S_W)}, 1")
        self.emit(f"s_lshl_b32 {sp(S_W)}, {sp(S_W)}, 8",
                  f"s_lshl_b32 {sp(S_Y)}, {sp(S_WAVE)}, 6",
                  f"s_add_u32 {sp(S_W)}, {sp(S_W)}, {sp(S_Y)}",
                  f"s_mov_b32 {sp(S_Y)}, 512")
        self.mul64(S_RO, S_RO + 1, S_W, S_Y)
        self.add64_to(S_RO, A_PO, S_RO, S_RO + 1)
        self.emit(f"s_mov_b32 {sp(S_Y)}, 4")
        self.mul64(S_RL, S_RL + 1, S_W, S_Y)
        self.add64_to(S_RL, A_PL, S_RL, S_RL + 1)
        self.emit(f"s_mov_b32 {sp(S_RO + 2)}, 32768", f"s_mov_b32 {sp(S_RO + 3)}, 0x20000",
                  f"s_mov_b32 {sp(S_RL + 2)}, 256", f"s_mov_b32 {sp(S_RL + 3)}, 0x20000")

    def merge2(self, which):
        """Complete stream `which` of a two-piece item: the other piece's
        partial from its slot, this piece's own part from its registers
        (normalised exactly as write_state stores it), combined in piece order
        with the same operations as merge(), so either piece gives the same
        bits. O, m, l and the weight sums are this piece's end state."""
        u = self.new_uid()
        T = V_T
        VL, INV, LSO = (T + 4, T + 5), (T + 6, T + 7), (T + 8, T + 9)
        VA, VB, VM, VI, VO = T + 10, T + 11, T + 12, T + 13, T + 14
        OUT = V_Y                                   # 64: one block's output rows
        other = S_GG
        # every P V and weight-sum MFMA has completed (O and the sums are read below)
        self.emit("s_nop 7", "s_nop 7", "s_nop 7")
        # the other segment, and whether this piece comes first
        self.emit(f"s_cmp_eq_u32 {sp(S_G)}, {sp(S_GLO)}",
                  f"s_cselect_b32 {sp(other)}, {sp(S_GHI)}, {sp(S_GLO)}")
        self.slot_resources(other, which)
        self.emit(f"v_and_b32_e32 {vp(T)}, 31, {vp(V_LANE)}",
                  f"v_lshrrev_b32_e32 {vp(T + 1)}, 5, {vp(V_LANE)}",
                  f"v_lshlrev_b32_e32 {vp(T + 1)}, 4, {vp(T + 1)}")
        for qb in range(2):
            # the other piece's rows 32 qb + ql: LSE and O (into the operand AGPRs)
            self.emit(f"v_add_u32_e32 {vp(T + 2)}, {32 * qb}, {vp(T)}",
                      f"v_lshlrev_b32_e32 {vp(T + 3)}, 2, {vp(T + 2)}",
                      f"v_lshl_add_u32 {vp(VO)}, {vp(T + 2)}, 9, {vp(T + 1)}",
                      "s_nop 1",
                      f"buffer_load_dword {vp(VL[qb])}, {vp(T + 3)}, {sp(S_RL, 4)}, 0 offen sc1")
            for db in range(4):
                for j in range(4):
                    self.emit(f"buffer_load_dwordx4 {ap(64 * qb + 16 * db + 4 * j, 4)}, {vp(VO)}, {sp(S_RO, 4)}, 0 "
                              f"offen offset:{128 * db + 32 * j} sc1")
        # own part: 1 / (sum of the rounded weights), LSE = m scale + ln(l total)
        for qb in range(2):
            m, l = V_ST[qb], V_ST[qb] + 3
            if NORM == "mfma":
                self.emit(f"v_accvgpr_read_b32 {vp(INV[qb])}, {ap(A_LR[qb])}")
            elif NORM == "mfma16":
                self.emit(*self.lr16(qb, INV[qb], T + 3, T + 2))
            elif NORM == "valu":
                self.emit(f"v_mov_b32_e32 {vp(INV[qb])}, {vp(V_ST[qb] + 1)}", f"v_mov_b32_e32 {vp(T + 3)}, {vp(V_ST[qb] + 1)}",
                          "s_nop 1",
                          f"v_permlane32_swap_b32 {vp(INV[qb])}, {vp(T + 3)}",
                          "s_nop 1",
                          f"v_add_f32_e32 {vp(INV[qb])}, {vp(INV[qb])}, {vp(T + 3)}")
            self.emit(f"v_mov_b32_e32 {vp(T + 2)}, {vp(l)}", f"v_mov_b32_e32 {vp(T + 3)}, {vp(l)}",
                      "s_nop 1",
                      f"v_permlane32_swap_b32 {vp(T + 2)}, {vp(T + 3)}",
                      "s_nop 1",
                      f"v_add_f32_e32 {vp(T + 2)}, {vp(T + 2)}, {vp(T + 3)}")
            if NORM == "fp32":
                self.emit(f"v_mov_b32_e32 {vp(INV[qb])}, {vp(T + 2)}")
            self.emit(f"v_rcp_f32_e32 {vp(INV[qb])}, {vp(INV[qb])}",
                      f"v_log_f32_e32 {vp(T + 2)}, {vp(T + 2)}",
                      "s_nop 1",
                      f"v_mul_f32_e32 {vp(T + 2)}, 0x3f317218, {vp(T + 2)}",
                      f"v_fma_f32 {vp(LSO[qb])}, {vp(m)}, {sp(A_SCALE)}, {vp(T + 2)}")
        self.emit("s_waitcnt vmcnt(0)")
        self.row_resources(which)
        self.emit(f"v_lshrrev_b32_e32 {vp(T + 1)}, 5, {vp(V_LANE)}",
                  f"v_cmp_ne_u32_e32 vcc, 0, {vp(T + 1)}",
                  f"v_lshlrev_b32_e32 {vp(T + 1)}, 4, {vp(T + 1)}",
                  f"s_cmp_eq_u32 {sp(S_G)}, {sp(S_GLO)}",
                  f"s_cbranch_scc0 .Lm2_second{u}")
        for own_first in (True, False):
            if not own_first:
                self.emit(f".Lm2_second{u}:")
            for qb in range(2):
                L1, L2 = (LSO[qb], VL[qb]) if own_first else (VL[qb], LSO[qb])
                self.emit(f"v_max_f32_e32 {vp(VM)}, {vp(L1)}, {vp(L2)}",
                          f"v_sub_f32_e32 {vp(VA)}, {vp(L1)}, {vp(VM)}",
                          f"v_sub_f32_e32 {vp(VB)}, {vp(L2)}, {vp(VM)}",
                          f"v_mul_f32_e32 {vp(VA)}, 0x3fb8aa3b, {vp(VA)}",
                          f"v_mul_f32_e32 {vp(VB)}, 0x3fb8aa3b, {vp(VB)}",
                          f"v_exp_f32_e32 {vp(VA)}, {vp(VA)}",
                          f"v_exp_f32_e32 {vp(VB)}, {vp(VB)}",
                          "s_nop 1",
                          f"v_add_f32_e32 {vp(VI)}, {vp(VA)}, {vp(VB)}",
                          "s_nop 1",
                          f"v_log_f32_e32 {vp(T + 2)}, {vp(VI)}",
                          f"v_rcp_f32_e32 {vp(VI)}, {vp(VI)}",
                          f"v_and_b32_e32 {vp(T)}, 31, {vp(V_LANE)}",
                          f"v_add_u32_e32 {vp(T)}, {32 * qb}, {vp(T)}",
                          f"v_mul_lo_u32 {vp(VO)}, {vp(T)}, {sp(S_X)}",
                          f"v_add_u32_e32 {vp(VO)}, {vp(VO)}, {vp(T + 1)}",       # O voffset
                          "s_nop 1")
                for i in range(64):
                    own, oth, acc = T + 3, T + 15, OUT + i
                    self.emit(f"v_mul_f32_e32 {vp(own)}, {vp(INV[qb])}, {vp(V_O[qb] + i)}",
                              f"v_accvgpr_read_b32 {vp(oth)}, {ap(64 * qb + i)}")
                    x1, x2 = (own, oth) if own_first else (oth, own)
                    self.emit(f"v_mul_f32_e32 {vp(acc)}, {vp(x1)}, {vp(VA)}",
                              f"v_fmac_f32_e32 {vp(acc)}, {vp(VB)}, {vp(x2)}",
                              f"v_mul_f32_e32 {vp(acc)}, {vp(VI)}, {vp(acc)}")
                for db in range(4):
                    for j in range(4):
                        self.emit(f"buffer_store_dwordx4 {vp(OUT + 16 * db + 4 * j, 4)}, {vp(VO)}, {sp(S_RO, 4)}, 0 "
                                  f"offen offset:{128 * db + 32 * j}")
                self.emit(f"v_fmac_f32_e32 {vp(VM)}, 0x3f317218, {vp(T + 2)}",
                          f"v_lshlrev_b32_e32 {vp(T)}, 2, {vp(T)}",
                          f"v_mov_b32_e32 {vp(T + 2)}, 0x40000000",
                          "s_nop 1",
                          f"v_cndmask_b32_e32 {vp(T)}, {vp(T)}, {vp(T + 2)}, vcc",
                          "s_nop 1",
                          f"buffer_store_dword {vp(VM)}, {vp(T)}, {sp(S_RL, 4)}, 0 offen",
                          "s_waitcnt vmcnt(0)")
            if own_first:
                self.emit(f"s_branch .Lm2_done{u}")
        self.emit(f".Lm2_done{u}:")

    def merge(self, which):
        """Complete stream `which` of this item from every piece's partial
        (this wave's 64 rows, both 32-row blocks per round trip): online
        Eq. 11-12 in piece order, then the normalised rows and LSE to the
        output. O, the score and operand registers are free here (the piece
        has ended): block 0 accumulates in O's first half and loads into its
        second, block 1 accumulates in the score registers and loads into the
        Q operand registers."""
        u = self.new_uid()
        T = V_T
        ACC = (V_O[0], V_Y)                 # 64 each: accumulators of blocks 0 / 1
        BUF = (V_O[1], A_Q[0])              # 64 each: a piece's rows (block 1 in AGPRs)
        VM, VS, VL, VOL, VOO = ((T + 4, T + 5), (T + 6, T + 7), (T + 8, T + 9), (T + 10, T + 11), (T + 12, T + 13))
        VA, VB = T + 14, T + 15
        self.piece_segments(which)
        # lane offsets in a slot: row 32 qb + ql; O bytes 16 hh within the row
        self.emit(f"v_and_b32_e32 {vp(T)}, 31, {vp(V_LANE)}",
                  f"v_lshrrev_b32_e32 {vp(T + 1)}, 5, {vp(V_LANE)}",
                  f"v_lshlrev_b32_e32 {vp(T + 1)}, 4, {vp(T + 1)}")
        for qb in range(2):
            self.emit(f"v_add_u32_e32 {vp(T + 2)}, {32 * qb}, {vp(T)}",
                      f"v_lshlrev_b32_e32 {vp(VOL[qb])}, 2, {vp(T + 2)}",
                      f"v_lshl_add_u32 {vp(VOO[qb])}, {vp(T + 2)}, 9, {vp(T + 1)}",
                      f"v_mov_b32_e32 {vp(VM[qb])}, 0xff800000",
                      f"v_mov_b32_e32 {vp(VS[qb])}, 0")
            for i in range(64):
                self.emit(f"v_mov_b32_e32 {vp(ACC[qb] + i)}, 0")
        self.emit(f"s_mov_b32 {sp(S_GG)}, {sp(S_GLO)}",
                  f".Lmg{u}:")
        self.slot_resources(S_GG, which)
        for qb in range(2):
            self.emit(f"buffer_load_dword {vp(VL[qb])}, {vp(VOL[qb])}, {sp(S_RL, 4)}, 0 offen sc1")
            reg = vp if qb == 0 else ap
            for db in range(4):
                for j in range(4):
                    self.emit(f"buffer_load_dwordx4 {reg(BUF[qb] + 16 * db + 4 * j, 4)}, {vp(VOO[qb])}, "
                              f"{sp(S_RO, 4)}, 0 offen offset:{128 * db + 32 * j} sc1")
        self.emit("s_waitcnt vmcnt(0)")
        for qb in range(2):
            # m' = max(m, l); a = e^(m - m'), b = e^(l - m'); acc = a acc + b o; s = a s + b
            self.emit(f"v_max_f32_e32 {vp(T)}, {vp(VM[qb])}, {vp(VL[qb])}",
                      f"v_sub_f32_e32 {vp(VA)}, {vp(VM[qb])}, {vp(T)}",
                      f"v_sub_f32_e32 {vp(VB)}, {vp(VL[qb])}, {vp(T)}",
                      f"v_mov_b32_e32 {vp(VM[qb])}, {vp(T)}",
                      f"v_mul_f32_e32 {vp(VA)}, 0x3fb8aa3b, {vp(VA)}",
                      f"v_mul_f32_e32 {vp(VB)}, 0x3fb8aa3b, {vp(VB)}",
                      f"v_exp_f32_e32 {vp(VA)}, {vp(VA)}",
                      f"v_exp_f32_e32 {vp(VB)}, {vp(VB)}",
                      "s_nop 1",
                      f"v_mul_f32_e32 {vp(VS[qb])}, {vp(VS[qb])}, {vp(VA)}",
                      f"v_add_f32_e32 {vp(VS[qb])}, {vp(VS[qb])}, {vp(VB)}")
            for i in range(64):
                acc = ACC[qb] + i
                if qb == 0:
                    src = BUF[0] + i
                else:
                    src = T + 2 + (i & 1)
                    self.emit(f"v_accvgpr_read_b32 {vp(src)}, {ap(BUF[1] + i)}")
                self.emit(f"v_mul_f32_e32 {vp(acc)}, {vp(acc)}, {vp(VA)}",
                          f"v_fmac_f32_e32 {vp(acc)}, {vp(VB)}, {vp(src)}")
        self.emit(f"s_add_u32 {sp(S_GG)}, {sp(S_GG)}, 1",
                  f"s_cmp_le_u32 {sp(S_GG)}, {sp(S_GHI)}",
                  f"s_cbranch_scc1 .Lmg{u}")
        # the completed rows: O = acc / s, LSE = m + ln s (lanes of the lower half)
        self.row_resources(which)
        self.emit(f"v_and_b32_e32 {vp(T)}, 31, {vp(V_LANE)}",
                  f"v_lshrrev_b32_e32 {vp(T + 1)}, 5, {vp(V_LANE)}",
                  f"v_lshlrev_b32_e32 {vp(T + 2)}, 4, {vp(T + 1)}",
                  f"v_cmp_ne_u32_e32 vcc, 0, {vp(T + 1)}",
                  f"v_mov_b32_e32 {vp(T + 1)}, 0x40000000")
        for qb in range(2):
            self.emit(f"v_rcp_f32_e32 {vp(VA)}, {vp(VS[qb])}",
                      f"v_add_u32_e32 {vp(T + 3)}, {32 * qb}, {vp(T)}",
                      f"v_mul_lo_u32 {vp(VB)}, {vp(T + 3)}, {sp(S_X)}",
                      f"v_add_u32_e32 {vp(VB)}, {vp(VB)}, {vp(T + 2)}",         # O voffset
                      "s_nop 1")
            for i in range(64):
                self.emit(f"v_mul_f32_e32 {vp(ACC[qb] + i)}, {vp(VA)}, {vp(ACC[qb] + i)}")
            for db in range(4):
                for j in range(4):
                    self.emit(f"buffer_store_dwordx4 {vp(ACC[qb] + 16 * db + 4 * j, 4)}, {vp(VB)}, "
                              f"{sp(S_RO, 4)}, 0 offen offset:{128 * db + 32 * j}")
            self.emit(f"v_log_f32_e32 {vp(VL[qb])}, {vp(VS[qb])}",
                      f"v_lshlrev_b32_e32 {vp(T + 3)}, 2, {vp(T + 3)}",
                      "s_nop 1",
                      f"v_fmac_f32_e32 {vp(VM[qb])}, 0x3f317218, {vp(VL[qb])}",
                      f"v_cndmask_b32_e32 {vp(T + 3)}, {vp(T + 3)}, {vp(T + 1)}, vcc",
                      "s_nop 1",
                      f"buffer_store_dword {vp(VM[qb])}, {vp(T + 3)}, {sp(S_RL, 4)}, 0 offen")
        self.emit("s_waitcnt vmcnt(0)")

    # ---------------------------------------------------------------- tile loop
    def prologue(self, b):
        """Restart of the compute pipeline at tile t (ring buffer b): the K
        operands of its first half are in registers. Its block-0 softmax step
        is resolved by the first phase of the tile body."""
        self.label(f".Lpro{b}")
        self.emit("s_waitcnt lgkmcnt(0)")
        for i in self.mfma_scores(V_Y, V_Z[0]):
            self.emit(i)
        self.emit("s_nop 7")
        for i in self.lds_k(b, 1):
            self.emit(i)
        self.emit("s_nop 7", "s_nop 7", "s_nop 7")
        body, check = self.softmax(0, V_Y, V_P0[0], S_NV + b, 0)
        for i in body + check:
            self.emit(i)
        self.emit(f"s_branch .Ltile{b}")

    def tile_body(self, B):
        """Tile t in ring buffer B. Each softmax step's trigger is resolved
        after the first matrix instruction of the following phase."""
        nb = (B + 1) & 3
        self.label(f".Ltile{B}")
        self.emit(f"s_sub_i32 {sp(S_BUDGET)}, {sp(S_BUDGET)}, 1",
                  f"s_cmp_lt_i32 {sp(S_BUDGET)}, 0",
                  "s_cbranch_scc1 .Lend")
        # A(2t): scores of half 2t+1 | softmax of half 2t, block 1 | V of half 2t
        # (resolves block 0's step of half 2t, from the prologue or B(2t-1))
        body, check = self.softmax(1, V_Z[0], V_P1, S_NV + B, 0)
        self.phase(self.mfma_scores(V_Y, V_Z[1]), self.lds_v(B, 0), body, check,
                   pre=self.resolve(0, V_Y, V_P0[0]))
        # barrier: tile t+1 resident everywhere; tile t-1's buffer is free
        # (every tile step issues the loads of one tile, so the loads of tile
        # t+2 are the only ones that may still be in flight)
        self.emit("s_waitcnt vmcnt(8)", "s_barrier", f"s_add_u32 {sp(S_X)}, {sp(S_T)}, 3")
        # B(2t): P V of half 2t | softmax of half 2t+1, block 0 | K of half 2t+2,
        # with the loads of tile t+3 into the buffer tile t-1 has left
        body, check = self.softmax(0, V_Y, V_P0[1], S_NV + B, 1)
        self.phase(self.mfma_pv(V_P0[0]), self.lds_k(nb, 0), body, check,
                   stage=self.stage_list(S_X, (B + 3) & 3), pre=self.resolve(1, V_Z[0], V_P1))
        self.emit(f"s_add_u32 {sp(S_X)}, {sp(S_T)}, 1",
                  f"s_cmp_eq_u32 {sp(S_X)}, {sp(S_FL)}",
                  f"s_cbranch_scc1 .Ltail{B}")
        # A(2t+1): scores of half 2t+2 | softmax of half 2t+1, block 1 | V of half 2t+1
        body, check = self.softmax(1, V_Z[1], V_P1, S_NV + B, 1)
        self.phase(self.mfma_scores(V_Y, V_Z[0]), self.lds_v(B, 1), body, check,
                   pre=self.resolve(0, V_Y, V_P0[1]))
        # B(2t+1): P V of half 2t+1 | softmax of half 2t+2, block 0 | K of half 2t+3
        body, check = self.softmax(0, V_Y, V_P0[0], S_NV + nb, 0)
        self.phase(self.mfma_pv(V_P0[1]), self.lds_k(nb, 1), body, check,
                   pre=self.resolve(1, V_Z[1], V_P1))
        self.emit(f"s_add_u32 {sp(S_T)}, {sp(S_T)}, 1")
        if B == 3:
            self.emit(".Ltile_wrap:", "s_branch .Ltile0")

    def tail(self, B):
        """Last half of tile t before a flush point: no scores of the next
        half, no softmax of the next half."""
        nb = (B + 1) & 3
        self.label(f".Ltail{B}")
        body, check = self.softmax(1, V_Z[1], V_P1, S_NV + B, 1)
        self.phase([], self.lds_v(B, 1), body, check + self.resolve(1, V_Z[1], V_P1),
                   pre=self.resolve(0, V_Y, V_P0[1]))
        self.phase(self.mfma_pv(V_P0[1]), [], [])
        self.emit(f"s_add_u32 {sp(S_T)}, {sp(S_T)}, 1",
                  f"s_cmp_eq_u32 {sp(S_T)}, {sp(S_TB)}",
                  "s_cbranch_scc1 .Lpiece_end")
        # dual-stream snapshot at the end of the local set: O, LSE of the
        # local keys, to the local output (piece from tile 0) or the slot
        u = self.new_uid()
        self.emit(f"s_cmp_eq_u32 {sp(S_TA)}, 0", f"s_cbranch_scc0 .Lsnap_slot{u}")
        self.write_state(True, 1)
        self.emit(f"s_branch .Lsnap_done{u}", f".Lsnap_slot{u}:")
        self.write_state(False, 1)
        self.publish(1)
        self.emit(f".Lsnap_done{u}:",
                  f"s_mov_b32 {sp(S_FL)}, {sp(S_TB)}",
                  f"s_branch .Lpro{nb}")

    # ---------------------------------------------------------------- kernel
    def lane_constants(self):
        T = V_T
        self.emit(f"v_and_b32_e32 {vp(V_LANE)}, 63, {vp(V_TID)}")
        # K operand addresses: row ql, chunk (2 kk + hh) ^ (ql & 15)
        self.emit(f"v_and_b32_e32 {vp(T)}, 31, {vp(V_LANE)}",            # ql
                  f"v_lshrrev_b32_e32 {vp(T + 1)}, 5, {vp(V_LANE)}",      # hh
                  f"v_and_b32_e32 {vp(T + 2)}, 15, {vp(V_LANE)}")        # ql & 15
        for kk in range(8):
            self.emit(f"v_add_u32_e32 {vp(T + 3)}, {2 * kk}, {vp(T + 1)}",
                      f"v_xor_b32_e32 {vp(T + 3)}, {vp(T + 3)}, {vp(T + 2)}",
                      f"v_lshlrev_b32_e32 {vp(T + 3)}, 4, {vp(T + 3)}",
                      f"v_lshl_add_u32 {vp(V_KOFF + kk)}, {vp(T)}, 8, {vp(T + 3)}")
        # V transpose-read addresses: with sl = lane & 15, g1 = (lane >> 4) & 1:
        # row = 8 h2 + 4 hh + (sl >> 2), chunk = 4 db + 2 g1 + ((sl & 3) >> 1),
        # swizzle = 4 (sl >> 2) ^ 2 hh, plus 8 bytes for odd sl
        self.emit(f"v_and_b32_e32 {vp(T + 2)}, 15, {vp(V_LANE)}",        # sl
                  f"v_lshrrev_b32_e32 {vp(T + 3)}, 2, {vp(T + 2)}",      # sl >> 2
                  f"v_bfe_u32 {vp(T + 4)}, {vp(V_LANE)}, 4, 1",          # g1
                  f"v_bfe_u32 {vp(T + 5)}, {vp(T + 2)}, 1, 1",           # (sl & 3) >> 1
                  f"v_and_b32_e32 {vp(T + 6)}, 1, {vp(T + 2)}",
                  f"v_lshlrev_b32_e32 {vp(T + 6)}, 3, {vp(T + 6)}",      # 8 (sl & 1)
                  f"v_lshlrev_b32_e32 {vp(T + 7)}, 2, {vp(T + 3)}",
                  f"v_lshlrev_b32_e32 {vp(T + 8)}, 1, {vp(T + 1)}",
                  f"v_xor_b32_e32 {vp(T + 7)}, {vp(T + 7)}, {vp(T + 8)}",  # swizzle
                  f"v_lshlrev_b32_e32 {vp(T + 8)}, 2, {vp(T + 1)}",
                  f"v_add_u32_e32 {vp(T + 8)}, {vp(T + 8)}, {vp(T + 3)}",   # 4 hh + (sl >> 2)
                  f"v_lshlrev_b32_e32 {vp(T + 9)}, 1, {vp(T + 4)}",
                  f"v_add_u32_e32 {vp(T + 9)}, {vp(T + 9)}, {vp(T + 5)}")   # 2 g1 + ((sl & 3) >> 1)
        for h2 in range(2):
            for db in range(4):
                r = V_VADDR + 4 * h2 + db
                self.emit(f"v_add_u32_e32 {vp(T + 10)}, {8 * h2}, {vp(T + 8)}",          # row
                          f"v_add_u32_e32 {vp(T + 11)}, {4 * db}, {vp(T + 9)}",          # chunk
                          f"v_xor_b32_e32 {vp(T + 11)}, {vp(T + 11)}, {vp(T + 7)}",
                          f"v_lshlrev_b32_e32 {vp(T + 11)}, 4, {vp(T + 11)}",
                          f"v_lshl_add_u32 {vp(r)}, {vp(T + 10)}, 8, {vp(T + 11)}",
                          f"v_add_u32_e32 {vp(r)}, {vp(r)}, {vp(T + 6)}",
                          f"v_add_u32_e32 {vp(r)}, 0x{V_REGION:x}, {vp(r)}")
        # staging voffsets of lane l of wave w, load q: row = 16 w + 4 q + (l >> 4),
        # stored chunk st = l & 15; K: chunk st ^ (row & 15) = st ^ (4 q + (l >> 4)),
        # V: st ^ (4 (row & 3) ^ 2 ((row >> 2) & 1)) = st ^ (4 (l >> 4) ^ 2 (q & 1));
        # less the load's instruction offset 1024 q
        self.emit(f"v_lshrrev_b32_e32 {vp(T)}, 4, {vp(V_LANE)}",         # l >> 4
                  f"v_and_b32_e32 {vp(T + 1)}, 15, {vp(V_LANE)}",        # st
                  f"s_lshl_b32 {sp(S_X)}, {sp(S_WAVE)}, 4",
                  f"v_add_u32_e32 {vp(T + 4)}, {sp(S_X)}, {vp(T)}",      # 16 w + (l >> 4)
                  f"v_lshlrev_b32_e32 {vp(T + 5)}, 2, {vp(T)}")          # 4 (l >> 4)
        for q in range(4):
            self.emit(f"v_add_u32_e32 {vp(T + 6)}, {4 * q}, {vp(T + 4)}",          # row
                      f"v_mul_lo_u32 {vp(T + 6)}, {vp(T + 6)}, {sp(A_LD2)}",
                      f"v_subrev_u32_e32 {vp(T + 6)}, {1024 * q}, {vp(T + 6)}",    # row bytes - 1024 q
                      f"v_add_u32_e32 {vp(T + 2)}, {4 * q}, {vp(T)}",
                      f"v_xor_b32_e32 {vp(T + 2)}, {vp(T + 2)}, {vp(T + 1)}",
                      f"v_lshl_add_u32 {vp(V_STK + q)}, {vp(T + 2)}, 4, {vp(T + 6)}",
                      f"v_xor_b32_e32 {vp(T + 3)}, {2 * (q & 1)}, {vp(T + 5)}",
                      f"v_xor_b32_e32 {vp(T + 3)}, {vp(T + 3)}, {vp(T + 1)}",
                      f"v_lshl_add_u32 {vp(V_STV + q)}, {vp(T + 3)}, 4, {vp(T + 6)}")
        # Q load voffsets: row (32 qb + ql), bytes 16 hh within the head's slice
        self.emit(f"v_and_b32_e32 {vp(T)}, 31, {vp(V_LANE)}",
                  f"v_lshrrev_b32_e32 {vp(T + 1)}, 5, {vp(V_LANE)}",
                  f"v_lshlrev_b32_e32 {vp(T + 1)}, 4, {vp(T + 1)}")
        for qb in range(2):
            self.emit(f"v_add_u32_e32 {vp(T + 2)}, {32 * qb}, {vp(T)}",
                      f"v_mul_lo_u32 {vp(T + 2)}, {vp(T + 2)}, {sp(A_LD2)}",
                      f"v_add_u32_e32 {vp(V_QOFF + qb)}, {vp(T + 2)}, {vp(T + 1)}")

    def piece_start(self):
        """Set up a piece: slot, head, Q operands, fresh state, the first
        three tiles staged, the K operands of the first half read."""
        T = V_T
        self.label(".Lpiece")
        # ta, tb, slot, head, qtile, hoff
        self.emit(f"s_mul_i32 {sp(S_X)}, {sp(S_ITEM)}, {sp(A_T)}",
                  f"s_sub_i32 {sp(S_TA)}, {sp(S_U0)}, {sp(S_X)}",
                  f"s_max_i32 {sp(S_TA)}, {sp(S_TA)}, 0",
                  f"s_sub_i32 {sp(S_TB)}, {sp(S_U1)}, {sp(S_X)}",
                  f"s_min_i32 {sp(S_TB)}, {sp(S_TB)}, {sp(A_T)}",
                  f"s_cmp_ge_i32 {sp(S_TA)}, {sp(S_TB)}",
                  "s_cbranch_scc1 .Lnext_item",
                  f"s_mul_i32 {sp(S_SLOT)}, {sp(S_G)}, {sp(A_MAXP)}",
                  f"s_add_u32 {sp(S_SLOT)}, {sp(S_SLOT)}, {sp(S_ITEM)}",
                  f"s_sub_u32 {sp(S_SLOT)}, {sp(S_SLOT)}, {sp(S_IFIRST)}")
        self.udiv(S_HEAD, S_ITEM, A_QT)
        self.emit(f"s_mul_i32 {sp(S_X)}, {sp(S_HEAD)}, {sp(A_QT)}",
                  f"s_sub_u32 {sp(S_QTILE)}, {sp(S_ITEM)}, {sp(S_X)}",
                  f"s_lshl_b32 {sp(S_HOFF2)}, {sp(S_HEAD)}, 8",               # head * 128 * 2 bytes
                  f"s_lshl_b32 {sp(S_QROWB)}, {sp(S_QTILE)}, 8",
                  f"s_lshl_b32 {sp(S_X)}, {sp(S_WAVE)}, 6",
                  f"s_add_u32 {sp(S_QROWB)}, {sp(S_QROWB)}, {sp(S_X)}")        # first query row of this wave
        # flush point: the end of the local set when it falls inside the piece
        self.emit(f"s_mov_b32 {sp(S_FL)}, {sp(S_TB)}",
                  f"s_cmp_eq_u32 {sp(A_DUAL)}, 0",
                  "s_cbranch_scc1 .Lfl_done",
                  f"s_cmp_lt_i32 {sp(S_TA)}, {sp(A_LT)}",
                  "s_cbranch_scc0 .Lfl_done",
                  f"s_cmp_lt_i32 {sp(A_LT)}, {sp(S_TB)}",
                  f"s_cselect_b32 {sp(S_FL)}, {sp(A_LT)}, {sp(S_FL)}",
                  ".Lfl_done:")
        # every wave is done with the previous piece's LDS tiles
        self.emit("s_barrier")
        self.emit(f"s_mov_b32 {sp(S_T)}, {sp(S_TA)}")
        self.stage_init(S_T)
        self.stage(S_T, 0)
        # Q resource: rows of this wave that exist; the head's 256 bytes of each
        self.mul64(S_X, S_Y, S_QROWB, A_LD2)
        self.emit(f"s_add_u32 {sp(S_X)}, {sp(S_X)}, {sp(S_HOFF2)}", f"s_addc_u32 {sp(S_Y)}, {sp(S_Y)}, 0")
        self.add64_to(S_RQ, A_QPTR, S_X, S_Y)
        self.emit(f"s_sub_i32 {sp(S_W)}, {sp(A_NQ)}, {sp(S_QROWB)}",
                  f"s_min_i32 {sp(S_W)}, {sp(S_W)}, 64",
                  f"s_max_i32 {sp(S_W)}, {sp(S_W)}, 0",
                  f"s_mul_i32 {sp(S_RQ + 2)}, {sp(S_W)}, {sp(A_LD2)}",
                  f"s_mov_b32 {sp(S_RQ + 3)}, 0x20000")
        for qb in range(2):
            for kk in range(8):
                self.emit(f"buffer_load_dwordx4 {ap(A_Q[qb] + 4 * kk, 4)}, {vp(V_QOFF + qb)}, {sp(S_RQ, 4)}, 0 "
                          f"offen offset:{32 * kk}")
        self.emit(f"s_add_u32 {sp(S_X)}, {sp(S_T)}, 1")
        self.stage(S_X, 1)
        self.emit(f"s_add_u32 {sp(S_X)}, {sp(S_T)}, 2")
        self.stage(S_X, 2)
        # fresh softmax state and O: m = -inf, -m c = +inf, so the first
        # weights are inf (or NaN) and the first half sets the reference
        for qb in range(2):
            m, nmc, l, alpha = V_ST[qb], V_ST[qb] + 2, V_ST[qb] + 3, V_ST[qb] + 5
            self.emit(f"v_mov_b32_e32 {vp(m)}, 0xff800000", f"v_mov_b32_e32 {vp(nmc)}, 0x7f800000",
                      f"v_mov_b32_e32 {vp(l)}, 0", f"v_mov_b32_e32 {vp(alpha)}, 1.0",
                      f"v_mov_b32_e32 {vp(V_ST[qb] + 1)}, 0")
            for i in range(64):
                self.emit(f"v_mov_b32_e32 {vp(V_O[qb] + i)}, 0")
        self.emit(f"v_mov_b32_e32 {vp(V_T)}, 0")
        for qb in range(2 if SUMS_ON_MFMA else 0):
            for i in range(N_LR):
                self.emit(f"v_accvgpr_write_b32 {ap(A_LR[qb] + i)}, {vp(V_T)}")
        # wait for tile ta and Q (the loads of tiles ta+1, ta+2 may stay in flight)
        self.emit("s_waitcnt vmcnt(16)", "s_barrier")
        for i in self.lds_k(0, 0):
            self.emit(i)
        self.emit("s_branch .Lpro0")

    def piece_end(self):
        self.label(".Lpiece_end")
        # end state: to the output rows when the piece is the whole item
        self.emit(f"s_cmp_eq_u32 {sp(S_TA)}, 0", "s_cbranch_scc0 .Lpe_slot",
                  f"s_cmp_eq_u32 {sp(S_TB)}, {sp(A_T)}", "s_cbranch_scc0 .Lpe_slot")
        self.write_state(True, 0)
        self.emit("s_branch .Lpe_local", ".Lpe_slot:")
        self.finish_stream(0)
        self.label(".Lpe_local")
        # a piece that ends inside (or at the end of) the local set also holds
        # its local result
        self.emit(f"s_cmp_eq_u32 {sp(A_DUAL)}, 0", "s_cbranch_scc1 .Lmerges",
                  f"s_cmp_le_i32 {sp(S_TB)}, {sp(A_LT)}", "s_cbranch_scc0 .Lmerges",
                  f"s_cmp_eq_u32 {sp(S_TA)}, 0", "s_cbranch_scc0 .Lpl_slot",
                  f"s_cmp_eq_u32 {sp(S_TB)}, {sp(A_LT)}", "s_cbranch_scc0 .Lpl_slot")
        self.write_state(True, 1)
        self.emit("s_branch .Lmerges", ".Lpl_slot:")
        self.finish_stream(1)
        # the streams this piece completes (one of them may have been counted at
        # the local snapshot inside the piece)
        self.label(".Lmerges")
        for which in range(2):
            self.emit(f"s_and_b32 {sp(S_X)}, {sp(S_MFLAG)}, {1 << which}",
                      f"s_cbranch_scc0 .Lmerged{which}")
            self.merge(which)
            self.label(f".Lmerged{which}")
        self.emit(f"s_mov_b32 {sp(S_MFLAG)}, 0")
        self.label(".Lnext_item")
        self.emit(f"s_sub_i32 {sp(S_ITEM)}, {sp(S_ITEM)}, 1",
                  f"s_cmp_ge_i32 {sp(S_ITEM)}, {sp(S_IFIRST)}",
                  "s_cbranch_scc1 .Lpiece",
                  "s_branch .Lend")

    def kernel(self):
        self.emit(f"s_load_dwordx16 {sp(S_ARG, 16)}, s[0:1], 0x0",
                  f"s_load_dwordx16 {sp(S_ARG + 16, 16)}, s[0:1], 0x40",
                  f"s_load_dwordx16 {sp(S_ARG + 32, 16)}, s[0:1], 0x80",
                  f"v_lshrrev_b32_e32 {vp(V_T)}, 6, {vp(V_TID)}",
                  "s_nop 1",
                  f"v_readfirstlane_b32 {sp(S_WAVE)}, {vp(V_T)}",
                  "s_waitcnt lgkmcnt(0)",
                  f"s_mov_b32 {sp(S_MFLAG)}, 0",
                  f"s_lshl_b32 {sp(S_WAVE4K)}, {sp(S_WAVE)}, 12",
                  # staging constants: records = nv * 2 ld + 256 - 2 ld, 64 rows = 128 ld bytes,
                  # the resources' format words
                  f"s_sub_i32 {sp(S_REC0)}, 0x100, {sp(A_LD2)}",
                  f"s_lshl_b32 {sp(S_LD128)}, {sp(A_LD2)}, 6",
                  f"s_mov_b32 {sp(S_RK + 3)}, 0x20000",
                  f"s_mov_b32 {sp(S_RV + 3)}, 0x20000",
                  # XCD-aware workgroup index
                  f"s_and_b32 {sp(S_X)}, s2, 7",
                  f"s_mul_i32 {sp(S_X)}, {sp(S_X)}, {sp(A_PERXCD)}",
                  f"s_lshr_b32 {sp(S_Y)}, s2, 3",
                  f"s_add_u32 {sp(S_G)}, {sp(S_X)}, {sp(S_Y)}",
                  f"s_cmp_ge_u32 {sp(S_G)}, {sp(A_NLOG)}",
                  "s_cbranch_scc1 .Lend",
                  f"s_cmp_eq_u32 {sp(A_NSEG)}, 0",
                  "s_cbranch_scc1 .Lnosplit",
                  f"s_mul_i32 {sp(S_Y)}, {sp(S_G)}, {sp(A_U)}")
        self.udiv(S_U0, S_Y, A_NSEG)
        self.emit(f"s_add_u32 {sp(S_Y)}, {sp(S_Y)}, {sp(A_U)}")
        self.udiv(S_U1, S_Y, A_NSEG)
        self.emit("s_branch .Lhave_u", ".Lnosplit:",
                  f"s_mul_i32 {sp(S_U0)}, {sp(S_G)}, {sp(A_T)}",
                  f"s_add_u32 {sp(S_U1)}, {sp(S_U0)}, {sp(A_T)}",
                  ".Lhave_u:")
        self.udiv(S_IFIRST, S_U0, A_T)
        self.emit(f"s_sub_u32 {sp(S_Y)}, {sp(S_U1)}, 1")
        self.udiv(S_ITEM, S_Y, A_T)
        self.emit(f"s_sub_u32 {sp(S_BUDGET)}, {sp(S_U1)}, {sp(S_U0)}",
                  f"s_add_u32 {sp(S_BUDGET)}, {sp(S_BUDGET)}, 16",
                  f"s_mov_b32 {sp(S_SLOT)}, 0")
        self.lane_constants()
        if NORM == "mfma16":
            # the selector: ones in lanes 0 and 32 (row 0, k-groups 0 and 2) and
            # 17 and 49 (row 1, k-groups 1 and 3), zeros elsewhere
            T = V_T
            self.emit(f"v_and_b32_e32 {vp(T + 1)}, 15, {vp(V_LANE)}",              # row m
                      f"v_bfe_u32 {vp(T + 2)}, {vp(V_LANE)}, 4, 1",                # k-group parity
                      f"v_xor_b32_e32 {vp(T + 2)}, {vp(T + 1)}, {vp(T + 2)}",
                      f"v_lshrrev_b32_e32 {vp(T + 1)}, 1, {vp(T + 1)}",
                      f"v_or_b32_e32 {vp(T + 2)}, {vp(T + 2)}, {vp(T + 1)}",       # 0: m < 2, m = parity
                      f"v_cmp_eq_u32_e32 vcc, 0, {vp(T + 2)}",
                      f"v_mov_b32_e32 {vp(T)}, 0x3f803f80",
                      "s_nop 1",
                      f"v_cndmask_b32_e32 {vp(T)}, 0, {vp(T)}, vcc")
        else:
            self.emit(f"v_mov_b32_e32 {vp(V_T)}, 0x3f803f80")
        for i in range(4 if SUMS_ON_MFMA else 0):
            self.emit(f"v_accvgpr_write_b32 {ap(A_ONES + i)}, {vp(V_T)}")
        self.piece_start()
        for b in range(4):
            self.prologue(b)
        for B in range(4):
            self.tile_body(B)
        for B in range(4):
            self.tail(B)
        self.piece_end()
        self.label(".Lend")
        self.emit("s_endpgm")
        for blk in self.ool:
            for i in blk:
                self.emit(i)

    def text(self):
        self.kernel()
        head = f"""\t.amdgcn_target "amdgcn-amd-amdhsa--gfx950"
\t.amdhsa_code_object_version 5
\t.text
\t.globl {KNAME}
\t.p2align 8
\t.type {KNAME},@function
{KNAME}:
"""
        body = "\n".join(self.lines)
        tail = f"""
\t.section .rodata,"a",@progbits
\t.p2align 6, 0x0
\t.amdhsa_kernel {KNAME}
\t\t.amdhsa_group_segment_fixed_size {LDS_BYTES}
\t\t.amdhsa_private_segment_fixed_size 0
\t\t.amdhsa_kernarg_size {ARGS_BYTES}
\t\t.amdhsa_user_sgpr_count 2
\t\t.amdhsa_user_sgpr_kernarg_segment_ptr 1
\t\t.amdhsa_system_sgpr_workgroup_id_x 1
\t\t.amdhsa_system_vgpr_workitem_id 0
\t\t.amdhsa_next_free_vgpr {256 + (N_AGPR + 7) // 8 * 8}
\t\t.amdhsa_next_free_sgpr 102
\t\t.amdhsa_accum_offset 256
\t\t.amdhsa_reserve_vcc 1
\t\t.amdhsa_float_denorm_mode_32 3
\t\t.amdhsa_float_denorm_mode_16_64 3
\t\t.amdhsa_dx10_clamp 1
\t\t.amdhsa_ieee_mode 1
\t.end_amdhsa_kernel
\t.amdgpu_metadata
---
amdhsa.kernels:
  - .agpr_count:     {N_AGPR}
    .args:
      - .offset:         0
        .size:           {ARGS_BYTES}
        .value_kind:     by_value
    .group_segment_fixed_size: {LDS_BYTES}
    .kernarg_segment_align: 8
    .kernarg_segment_size: {ARGS_BYTES}
    .max_flat_workgroup_size: 256
    .name:           {KNAME}
    .private_segment_fixed_size: 0
    .sgpr_count:     104
    .sgpr_spill_count: 0
    .symbol:         {KNAME}.kd
    .uniform_work_group_size: 1
    .vgpr_count:     {256 + (N_AGPR + 7) // 8 * 8}
    .vgpr_spill_count: 0
    .wavefront_size: 64
amdhsa.target:   amdgcn-amd-amdhsa--gfx950
amdhsa.version:
  - 1
  - 2
...
\t.end_amdgpu_metadata
"""
        return head + body + "\n" + tail


def generate():
    return Gen().text()


if __name__ == "__main__":
    sys.stdout.write(generate())
