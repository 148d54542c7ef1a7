"""Generates proj_fast.s: the gfx950 assembly of the L-Layer output projection
(Sec. 3.1 step 3 with Eq. 4, Y = A W_new, the weight in the linear-layer
layout W_lin = W_new^T [d_out, d_in]) for widths that are multiples of 256, in
two kernels: bf16 operands with fp32 accumulation, and the W8A8 form (Sec. 4)
with int8 codes, int32 accumulation and the dequantisation
y = (float(acc) * s_a[row]) * s_w[col].

Y = A W_lin^T contracts over the contiguous dimension of both operands, so a
lane's matrix operand (8 bf16 or 16 int8 consecutive k of one row) is one
16-byte LDS read. One workgroup of 4 waves (one per SIMD) per output tile of
256 rows x 256 columns; wave (wr, wc) owns the 128 x 128 quarter at rows
128 wr, columns 128 wc as 4 x 4 blocks of 32 x 32 in its 256 accumulation
registers, so each operand read feeds four matrix instructions (the C++
kernel's waves of 64 x 128 read 50% more LDS bytes per instruction).

A stage is 64 bytes of k (32 bf16 or 64 int8) of the tile's 256 A rows
(region A) and of its W rows (region B), each row 64 bytes with its four
16-byte chunks XOR-swizzled by (row / 4) mod 4, so that each 16-lane group of
a read (16 consecutive rows, one chunk) covers all 64 banks. Stages go HBM ->
LDS by buffer loads straight into LDS, in a ring of four (three ahead); rows
past the last one read as zero through the buffer records.

Per stage: phase 0 issues the matrix instructions of the first half of the
stage's k, the reads of the second half and the loads of stage s + 3; phase 1
issues a quarter of the second half's instructions, waits for stage s + 1 (its
own loads, then the barrier that makes everyone's visible and frees the buffer
that stage s + 4 will use), then the rest with the reads of stage s + 1.

Work: whole 256 x 256 tiles fill full rounds of the chip; when the tiles left
over would keep at most half of a last round busy, each of them is computed as
two 256 x 128 halves by two workgroups (waves of 128 x 64), so no round is
mostly idle and every output element is still summed by one workgroup in one
order. Tiles are taken four row panels at a time, column by column, and each
XCD gets a contiguous range of them, so the workgroups resident on an XCD
stream few distinct panels through its L2.

Run as a script it prints the assembly; build.py assembles it.
"""

ARGS_BYTES = 96

# kernel arguments (byte offsets)
ARG_A, ARG_W, ARG_SA, ARG_SW, ARG_Y = 0, 8, 16, 24, 32
ARG_N, ARG_LD, ARG_LDY, ARG_TM, ARG_TN = 40, 44, 48, 52, 56
ARG_NWHOLE, ARG_PERXCD, ARG_PERXCDH, ARG_NHALF, ARG_STEPS, ARG_YBF16 = 60, 64, 68, 72, 76, 80

S_ARG = 8                       # s[8:31]


def arg(off):
    return S_ARG + off // 4


A_A, A_W, A_SA, A_SW, A_Y = (arg(o) for o in (ARG_A, ARG_W, ARG_SA, ARG_SW, ARG_Y))
A_N, A_LD, A_LDY, A_TM, A_TN = (arg(o) for o in (ARG_N, ARG_LD, ARG_LDY, ARG_TM, ARG_TN))
A_NWHOLE, A_PERXCD, A_PERXCDH, A_NHALF, A_STEPS, A_YBF16 = (
    arg(o) for o in (ARG_NWHOLE, ARG_PERXCD, ARG_PERXCDH, ARG_NHALF, ARG_STEPS, ARG_YBF16))

# SGPRs
S_RA, S_RB, S_OUT, S_RS, S_RW = 32, 36, 40, 44, 48   # resources: A, W, Y, s_a, s_w
S_WAVE, S_M0A, S_M0H = 52, 53, 54   # wave, wave * 4096, wave * 2048 (LDS bases of its loads)
S_ITEM, S_TI, S_TJ, S_HALF = 55, 56, 57, 58        # item, tile row / column, half (-1: whole)
S_STEP, S_BUDGET, S_SLD = 59, 60, 61               # stages done, loop guard, next stage to load
S_K, S_GM, S_R0, S_T = 62, 63, 64, 65
S_X, S_Y, S_Z = 66, 67, 68
S_RECA, S_RECB = 69, 70                            # records of a loaded stage (A / W side)
S_EO = 72                                          # 16: epilogue row offsets of accumulator element r
N_SGPR = 88

# VGPRs
V_TID, V_LANE = 0, 1
V_RA = 2                        # 2: A-side read addresses, k half 0 / 1 of a stage
V_RB = 4                        # 2: W side, whole tiles
V_RBH = 6                       # 2: W side, half tiles
V_ST = 8                        # 4: staging voffsets, load q (A side; W side of whole tiles)
V_STH = 12                      # 2: W side of half tiles
V_OPS = (16, 48)                # operand sets X / Y: A blocks at +4 b, W blocks at +16 + 4 b
V_T = 80                        # temporaries
V_EOFF = (96, 112)              # 16 each: epilogue voffsets of the elements of a block, per value buffer
N_VGPR = 128
N_AGPR = 256

GROUP = 4                       # row panels per group of the work order
EARLY = 4                       # phase 1 issues 1 / EARLY of its MFMAs before the wait for the next stage

REGION_B = 65536
STAGE_BYTES = 16384             # one region's share of a stage: 256 rows x 64 bytes
LDS_BYTES = 131072


def sp(r, n=1):
    return f"s{r}" if n == 1 else f"s[{r}:{r + n - 1}]"


def vp(r, n=1):
    return f"v{r}" if n == 1 else f"v[{r}:{r + n - 1}]"


def ap(r, n=1):
    return f"a{r}" if n == 1 else f"a[{r}:{r + n - 1}]"


class Gen:
    def __init__(self, i8):
        self.i8 = i8
        self.name = "ispa_proj_fast_i8" if i8 else "ispa_proj_fast_bf16"
        self.pre = ".Li" if i8 else ".Lb"
        self.lines = []
        self.uid = 0

    def L(self, name):
        return f"{self.pre}_{name}"

    def new_uid(self):
        self.uid += 1
        return self.uid

    def emit(self, *ins):
        for i in ins:
            self.lines.append("  " + i if not i.endswith(":") else i)

    def label(self, name):
        self.lines.append(self.L(name) + ":")

    # ---------------------------------------------------------------- setup
    def decode_tile(self):
        """S_ITEM -> (S_TI, S_TJ): row panels GROUP at a time (the last group
        may hold fewer), within a group column by column."""
        k, gm, r0, t = S_K, S_GM, S_R0, S_T
        self.emit(f"s_mov_b32 {sp(k)}, {sp(S_ITEM)}", f"s_mov_b32 {sp(r0)}, 0",
                  f"s_mul_i32 {sp(t)}, {sp(A_TN)}, {GROUP}",                 # items of a full group
                  self.L("grp") + ":",
                  f"s_sub_i32 {sp(gm)}, {sp(A_TM)}, {sp(r0)}",
                  f"s_cmp_lt_i32 {sp(gm)}, {GROUP}",
                  f"s_cbranch_scc1 {self.L('grp_last')}",
                  f"s_cmp_lt_i32 {sp(k)}, {sp(t)}",
                  f"s_cbranch_scc1 {self.L('grp_full')}",
                  f"s_sub_i32 {sp(k)}, {sp(k)}, {sp(t)}",
                  f"s_add_i32 {sp(r0)}, {sp(r0)}, {GROUP}",
                  f"s_branch {self.L('grp')}",
                  self.L("grp_full") + ":",
                  f"s_mov_b32 {sp(gm)}, {GROUP}",
                  self.L("grp_last") + ":",
                  # tj = k / gm, ti = r0 + k % gm (gm <= GROUP: by subtraction)
                  f"s_mov_b32 {sp(S_TJ)}, 0",
                  self.L("dm") + ":",
                  f"s_cmp_lt_i32 {sp(k)}, {sp(gm)}",
                  f"s_cbranch_scc1 {self.L('dm_done')}",
                  f"s_sub_i32 {sp(k)}, {sp(k)}, {sp(gm)}",
                  f"s_add_i32 {sp(S_TJ)}, {sp(S_TJ)}, 1",
                  f"s_branch {self.L('dm')}",
                  self.L("dm_done") + ":",
                  f"s_add_i32 {sp(S_TI)}, {sp(r0)}, {sp(k)}")

    def lane_constants(self):
        T = V_T
        self.emit(f"v_and_b32_e32 {vp(V_LANE)}, 63, {vp(V_TID)}")
        # reads: lane l takes row r = l & 31 of a 32-row block and the chunk
        # 2 s + (l >> 5) of k half s; stored at r * 64 + ((chunk ^ swz(r)) << 4),
        # swz(r) = (r >> 2) & 3 (block and wave offsets are multiples of 16 rows)
        self.emit(f"v_and_b32_e32 {vp(T)}, 31, {vp(V_LANE)}",               # r
                  f"v_lshrrev_b32_e32 {vp(T + 1)}, 5, {vp(V_LANE)}",        # h
                  f"v_bfe_u32 {vp(T + 2)}, {vp(T)}, 2, 2",                  # swz(r)
                  f"v_lshlrev_b32_e32 {vp(T + 3)}, 6, {vp(T)}")             # 64 r
        # wave (wr, wc) = (wave >> 1, wave & 1): A rows 128 wr; W rows 128 wc
        # (whole tiles) or 64 wc (half tiles)
        self.emit(f"s_lshr_b32 {sp(S_X)}, {sp(S_WAVE)}, 1",
                  f"s_lshl_b32 {sp(S_X)}, {sp(S_X)}, 13",                   # 8192 wr
                  f"s_and_b32 {sp(S_Y)}, {sp(S_WAVE)}, 1",
                  f"s_lshl_b32 {sp(S_Z)}, {sp(S_Y)}, 12",
                  f"s_add_u32 {sp(S_Z)}, {sp(S_Z)}, {REGION_B}",            # half: 64K + 4096 wc
                  f"s_lshl_b32 {sp(S_Y)}, {sp(S_Y)}, 13",
                  f"s_add_u32 {sp(S_Y)}, {sp(S_Y)}, {REGION_B}")            # whole: 64K + 8192 wc
        for s in range(2):
            self.emit(f"v_add_u32_e32 {vp(T + 4)}, {2 * s}, {vp(T + 1)}",   # chunk
                      f"v_xor_b32_e32 {vp(T + 4)}, {vp(T + 4)}, {vp(T + 2)}",
                      f"v_lshl_add_u32 {vp(T + 4)}, {vp(T + 4)}, 4, {vp(T + 3)}",
                      f"v_add_u32_e32 {vp(V_RA + s)}, {sp(S_X)}, {vp(T + 4)}",
                      f"v_add_u32_e32 {vp(V_RB + s)}, {sp(S_Y)}, {vp(T + 4)}",
                      f"v_add_u32_e32 {vp(V_RBH + s)}, {sp(S_Z)}, {vp(T + 4)}")
        # staging: load q of wave w fills LDS rows R0 + 16 q + (l >> 2), stored
        # chunk l & 3, R0 = 64 w (256-row side) or 32 w (128-row side); global
        # chunk (l & 3) ^ ((l >> 4) & 3); voffset = row * ld + chunk * 16 - 1024 q
        # (the instruction offset 1024 q applies to the memory and the LDS address)
        self.emit(f"v_lshrrev_b32_e32 {vp(T)}, 2, {vp(V_LANE)}",            # l >> 2
                  f"v_bfe_u32 {vp(T + 1)}, {vp(V_LANE)}, 4, 2",
                  f"v_and_b32_e32 {vp(T + 2)}, 3, {vp(V_LANE)}",
                  f"v_xor_b32_e32 {vp(T + 1)}, {vp(T + 1)}, {vp(T + 2)}",
                  f"v_lshlrev_b32_e32 {vp(T + 1)}, 4, {vp(T + 1)}",         # chunk bytes
                  f"s_lshl_b32 {sp(S_X)}, {sp(S_WAVE)}, 6",
                  f"s_lshl_b32 {sp(S_Y)}, {sp(S_WAVE)}, 5")
        for q in range(4):
            self.emit(f"v_add_u32_e32 {vp(T + 3)}, {16 * q}, {vp(T)}",
                      f"v_add_u32_e32 {vp(T + 4)}, {sp(S_X)}, {vp(T + 3)}",
                      f"v_mul_lo_u32 {vp(T + 4)}, {vp(T + 4)}, {sp(A_LD)}",
                      f"v_add_u32_e32 {vp(T + 4)}, {vp(T + 4)}, {vp(T + 1)}",
                      f"v_subrev_u32_e32 {vp(V_ST + q)}, {1024 * q}, {vp(T + 4)}")
            if q < 2:
                self.emit(f"v_add_u32_e32 {vp(T + 4)}, {sp(S_Y)}, {vp(T + 3)}",
                          f"v_mul_lo_u32 {vp(T + 4)}, {vp(T + 4)}, {sp(A_LD)}",
                          f"v_add_u32_e32 {vp(T + 4)}, {vp(T + 4)}, {vp(T + 1)}",
                          f"v_subrev_u32_e32 {vp(V_STH + q)}, {1024 * q}, {vp(T + 4)}")

    # ---------------------------------------------------------------- staging
    def stage_list(self, buf, nbj):
        """The direct loads of stage S_SLD into ring buffer `buf` and the
        advance of both sides by one stage, as an instruction list; a stage
        at or past the last one loads nothing (no records: zero fill)."""
        ins = [f"s_cmp_lt_u32 {sp(S_SLD)}, {sp(A_STEPS)}",
               f"s_cselect_b32 {sp(S_RA + 2)}, {sp(S_RECA)}, 0",
               f"s_cselect_b32 {sp(S_RB + 2)}, {sp(S_RECB)}, 0",
               f"s_add_u32 m0, {sp(S_M0A)}, {buf * STAGE_BYTES}\n  s_nop 0"]
        ins += [f"buffer_load_dwordx4 {vp(V_ST + q)}, {sp(S_RA, 4)}, 0 offen offset:{1024 * q} lds" for q in range(4)]
        if nbj == 4:
            ins += [f"s_add_u32 m0, {sp(S_M0A)}, {REGION_B + buf * STAGE_BYTES}\n  s_nop 0"]
            ins += [f"buffer_load_dwordx4 {vp(V_ST + q)}, {sp(S_RB, 4)}, 0 offen offset:{1024 * q} lds"
                    for q in range(4)]
        else:
            ins += [f"s_add_u32 m0, {sp(S_M0H)}, {REGION_B + buf * STAGE_BYTES}\n  s_nop 0"]
            ins += [f"buffer_load_dwordx4 {vp(V_STH + q)}, {sp(S_RB, 4)}, 0 offen offset:{1024 * q} lds"
                    for q in range(2)]
        ins += [f"s_add_u32 {sp(S_RA)}, {sp(S_RA)}, 64\n  s_addc_u32 {sp(S_RA + 1)}, {sp(S_RA + 1)}, 0",
                f"s_add_u32 {sp(S_RB)}, {sp(S_RB)}, 64\n  s_addc_u32 {sp(S_RB + 1)}, {sp(S_RB + 1)}, 0",
                f"s_add_u32 {sp(S_SLD)}, {sp(S_SLD)}, 1"]
        return ins

    # ---------------------------------------------------------------- matrix work
    @staticmethod
    def reads(buf, half, ops, nbj):
        """The operand reads of k half `half` of a stage: 4 A blocks, nbj W blocks."""
        rb = V_RB if nbj == 4 else V_RBH
        out = []
        for b in range(4):
            out.append(f"ds_read_b128 {vp(ops + 4 * b, 4)}, {vp(V_RA + half)} offset:{buf * STAGE_BYTES + 2048 * b}")
        for b in range(nbj):
            out.append(f"ds_read_b128 {vp(ops + 16 + 4 * b, 4)}, {vp(rb + half)} offset:{buf * STAGE_BYTES + 2048 * b}")
        return out

    def mfmas(self, ops, nbj):
        """acc(ai, bj) += A_ai W_bj^T over one k half: 4 nbj independent accumulations."""
        op = "v_mfma_i32_32x32x32_i8" if self.i8 else "v_mfma_f32_32x32x16_bf16"
        out = []
        for ai in range(4):
            for bj in range(nbj):
                acc = ap(16 * (nbj * ai + bj), 16)
                out.append(f"{op} {acc}, {vp(ops + 4 * ai, 4)}, {vp(ops + 16 + 4 * bj, 4)}, {acc}")
        return out

    def interleave(self, mfma, other, start=0):
        """MFMAs with the other instructions spread evenly after them (from
        MFMA `start` on)."""
        n = len(mfma) - start
        per = -(-len(other) // n) if n > 0 else len(other)
        k = 0
        for i, m in enumerate(mfma):
            self.emit(m)
            if i >= start:
                for o in other[k:k + per]:
                    self.emit(o)
                k += per
        for o in other[k:]:
            self.emit(o)

    def loop(self, nbj, tag):
        """Prologue (stages 0..2 loaded, stage 0's first reads) and the ring of
        four stage bodies for tiles of 32 nbj columns per wave."""
        X, Y = V_OPS
        loads = 8 if nbj == 4 else 6                  # direct loads per wave per stage
        for b in range(3):
            for i in self.stage_list(b, nbj):
                self.emit(i)
        # stage 0 resident everywhere (the loads of stages 1, 2 may stay in flight)
        self.emit(f"s_waitcnt vmcnt({2 * loads})", "s_barrier")
        for i in self.reads(0, 0, X, nbj):
            self.emit(i)
        for B in range(4):
            nb = (B + 1) & 3
            self.label(f"{tag}{B}")
            self.emit(f"s_sub_i32 {sp(S_BUDGET)}, {sp(S_BUDGET)}, 1",
                      f"s_cmp_lt_i32 {sp(S_BUDGET)}, 0",
                      f"s_cbranch_scc1 {self.L('end')}",
                      "s_waitcnt lgkmcnt(0)")
            # phase 0: k half 0 | reads of half 1 (set Y; the MFMAs reading Y last
            # were issued a phase ago) | loads of stage s + 3 into buffer (B + 3) & 3
            other = self.reads(B, 1, Y, nbj) + self.stage_list((B + 3) & 3, nbj)
            self.interleave(self.mfmas(X, nbj), other, start=1)
            # phase 1: k half 1 (set Y) | wait for stage s + 1 | reads of its half 0 (set X)
            m = self.mfmas(Y, nbj)
            first = len(m) // EARLY
            self.emit("s_waitcnt lgkmcnt(0)")
            for i in m[:first]:
                self.emit(i)
            # every wave's loads of stage s + 1 have landed (at most the loads of
            # stages s + 2 and s + 3 are outstanding per wave) and every wave is
            # done with stage s - 1's buffer
            self.emit(f"s_waitcnt vmcnt({2 * loads})", "s_barrier")
            self.interleave(m[first:], self.reads(nb, 0, X, nbj), start=0)
            self.emit(f"s_add_u32 {sp(S_STEP)}, {sp(S_STEP)}, 1",
                      f"s_cmp_ge_u32 {sp(S_STEP)}, {sp(A_STEPS)}",
                      f"s_cbranch_scc1 {self.L(tag + '_done')}")
            if B == 3:
                self.emit(f"s_branch {self.L(tag + '0')}")

    # ---------------------------------------------------------------- epilogue
    def epilogue(self, nbj, tag):
        """Y rows of this wave's quarter (rows past n are not stored) from its
        accumulators: fp32 or bf16 (round to nearest even); the int8 form
        dequantises each value as (float(acc) * s_a[row]) * s_w[col] first."""
        T = V_T
        u = self.new_uid()
        self.label(tag + "_done")
        # every MFMA has completed before the accumulation registers are read
        self.emit("s_waitcnt vmcnt(0) lgkmcnt(0)", "s_nop 7", "s_nop 7", "s_nop 7")
        cols_w = 32 * nbj                                # columns per wave
        # S_Z: element bytes; S_X: rows of the tile left from this wave's first row
        self.emit(f"s_cmp_eq_u32 {sp(A_YBF16)}, 0",
                  f"s_cselect_b32 {sp(S_Z)}, 4, 2",
                  f"s_lshl_b32 {sp(S_X)}, {sp(S_TI)}, 8",
                  f"s_lshr_b32 {sp(S_Y)}, {sp(S_WAVE)}, 1",
                  f"s_lshl_b32 {sp(S_Y)}, {sp(S_Y)}, 7",
                  f"s_add_u32 {sp(S_X)}, {sp(S_X)}, {sp(S_Y)}",           # first row of the quarter
                  f"s_sub_i32 {sp(S_T)}, {sp(A_N)}, {sp(S_X)}",
                  f"s_min_i32 {sp(S_T)}, {sp(S_T)}, 128",
                  f"s_max_i32 {sp(S_T)}, {sp(S_T)}, 0",                   # rows to store
                  # Y resource: base = y + row0 * ldy + col0 * esize
                  f"s_mul_hi_u32 {sp(S_Y)}, {sp(S_X)}, {sp(A_LDY)}",
                  f"s_mul_i32 {sp(S_K)}, {sp(S_X)}, {sp(A_LDY)}",
                  f"s_add_u32 {sp(S_OUT)}, {sp(A_Y)}, {sp(S_K)}",
                  f"s_addc_u32 {sp(S_OUT + 1)}, {sp(A_Y + 1)}, {sp(S_Y)}",
                  f"s_lshl_b32 {sp(S_K)}, {sp(S_TJ)}, 8",
                  f"s_max_i32 {sp(S_Y)}, {sp(S_HALF)}, 0",
                  f"s_lshl_b32 {sp(S_Y)}, {sp(S_Y)}, 7",
                  f"s_add_u32 {sp(S_K)}, {sp(S_K)}, {sp(S_Y)}",           # first column of the tile
                  f"s_and_b32 {sp(S_Y)}, {sp(S_WAVE)}, 1",
                  f"s_mul_i32 {sp(S_Y)}, {sp(S_Y)}, {cols_w}",
                  f"s_add_u32 {sp(S_K)}, {sp(S_K)}, {sp(S_Y)}",           # first column of the quarter
                  f"s_mul_i32 {sp(S_Y)}, {sp(S_K)}, {sp(S_Z)}",
                  f"s_add_u32 {sp(S_OUT)}, {sp(S_OUT)}, {sp(S_Y)}",
                  f"s_addc_u32 {sp(S_OUT + 1)}, {sp(S_OUT + 1)}, 0",
                  f"s_mul_i32 {sp(S_OUT + 2)}, {sp(S_T)}, {sp(A_LDY)}",
                  f"s_mov_b32 {sp(S_OUT + 3)}, 0x20000")
        if self.i8:
            # s_a from the quarter's first row (rows past n read as zero), s_w
            # from its first column
            self.emit(f"s_lshl_b32 {sp(S_Y)}, {sp(S_X)}, 2",
                      f"s_add_u32 {sp(S_RS)}, {sp(A_SA)}, {sp(S_Y)}",
                      f"s_addc_u32 {sp(S_RS + 1)}, {sp(A_SA + 1)}, 0",
                      f"s_lshl_b32 {sp(S_RS + 2)}, {sp(S_T)}, 2",
                      f"s_mov_b32 {sp(S_RS + 3)}, 0x20000",
                      f"s_lshl_b32 {sp(S_Y)}, {sp(S_K)}, 2",
                      f"s_add_u32 {sp(S_RW)}, {sp(A_SW)}, {sp(S_Y)}",
                      f"s_addc_u32 {sp(S_RW + 1)}, {sp(A_SW + 1)}, 0",
                      f"s_mov_b32 {sp(S_RW + 2)}, {4 * cols_w}",
                      f"s_mov_b32 {sp(S_RW + 3)}, 0x20000")
        # accumulator element r of lane l: row 8 (r >> 2) + 4 (l >> 5) + (r & 3), column l & 31
        for r in range(16):
            self.emit(f"s_mul_i32 {sp(S_EO + r)}, {sp(A_LDY)}, {8 * (r >> 2) + (r & 3)}")
        self.emit(f"v_lshrrev_b32_e32 {vp(T)}, 5, {vp(V_LANE)}",
                  f"v_lshlrev_b32_e32 {vp(T)}, 2, {vp(T)}",                  # 4 (l >> 5)
                  f"v_mul_lo_u32 {vp(T + 1)}, {vp(T)}, {sp(A_LDY)}",
                  f"v_and_b32_e32 {vp(T + 2)}, 31, {vp(V_LANE)}",
                  f"v_mul_lo_u32 {vp(T + 3)}, {vp(T + 2)}, {sp(S_Z)}",
                  f"v_add_u32_e32 {vp(T + 1)}, {vp(T + 1)}, {vp(T + 3)}")    # lane's voffset in a block
        if self.i8:
            self.emit(f"v_lshlrev_b32_e32 {vp(T + 4)}, 2, {vp(T)}",          # s_a: 4 (4 (l >> 5)) bytes
                      f"v_lshlrev_b32_e32 {vp(T + 5)}, 2, {vp(T + 2)}")      # s_w: 4 (l & 31)
        VB = (V_OPS[0], V_OPS[0] + 16)                                      # value buffers
        VSA, VSW = V_OPS[1], V_OPS[1] + 16                                  # int8: row / column scales
        if self.i8:
            for bj in range(nbj):
                self.emit(f"buffer_load_dword {vp(VSW + bj)}, {vp(T + 5)}, {sp(S_RW, 4)}, 0 offen offset:{128 * bj}")
        for bf in range(2):
            if bf == 0:
                self.emit(f"s_cmp_eq_u32 {sp(A_YBF16)}, 0", f"s_cbranch_scc0 {self.L(f'ybf{u}')}")
            else:
                self.label(f"ybf{u}")
            k = 0
            for ai in range(4):
                if self.i8:
                    # the 16 row scales of block row ai (the previous block row's
                    # stores may still be in flight; they do not use these registers)
                    for r in range(16):
                        self.emit(f"buffer_load_dword {vp(VSA + r)}, {vp(T + 4)}, {sp(S_RS, 4)}, 0 offen "
                                  f"offset:{4 * (32 * ai + 8 * (r >> 2) + (r & 3))}")
                    self.emit("s_waitcnt vmcnt(0)")
                for bj in range(nbj):
                    acc = 16 * (nbj * ai + bj)
                    buf = VB[k & 1]
                    if k >= 2:
                        # this buffer's stores (two blocks ago) have read their data and voffsets
                        self.emit("s_waitcnt vmcnt(16)")
                    # the element offsets go whole into the voffsets: the buffer
                    # records (rows that exist) bound voffset + instruction offset
                    vo = V_EOFF[k & 1]
                    self.emit(f"s_mul_i32 {sp(S_Y)}, {sp(A_LDY)}, {32 * ai}",
                              f"s_mul_i32 {sp(S_R0)}, {sp(S_Z)}, {32 * bj}",
                              f"s_add_u32 {sp(S_Y)}, {sp(S_Y)}, {sp(S_R0)}",
                              f"v_add_u32_e32 {vp(T + 6)}, {sp(S_Y)}, {vp(T + 1)}")
                    for r in range(16):
                        self.emit(f"v_add_u32_e32 {vp(vo + r)}, {sp(S_EO + r)}, {vp(T + 6)}")
                    for r in range(16):
                        self.emit(f"v_accvgpr_read_b32 {vp(buf + r)}, {ap(acc + r)}")
                    if self.i8:
                        for r in range(16):
                            self.emit(f"v_cvt_f32_i32_e32 {vp(buf + r)}, {vp(buf + r)}",
                                      f"v_mul_f32_e32 {vp(buf + r)}, {vp(buf + r)}, {vp(VSA + r)}",
                                      f"v_mul_f32_e32 {vp(buf + r)}, {vp(buf + r)}, {vp(VSW + bj)}")
                    if bf:
                        for r in range(16):
                            self.emit(f"v_cvt_pk_bf16_f32 {vp(buf + r)}, {vp(buf + r)}, {vp(buf + r)}")
                    self.emit("s_nop 1")
                    st = "buffer_store_short" if bf else "buffer_store_dword"
                    for r in range(16):
                        self.emit(f"{st} {vp(buf + r)}, {vp(vo + r)}, {sp(S_OUT, 4)}, 0 offen")
                    k += 1
            self.emit(f"s_branch {self.L(tag + '_stored')}")
        self.label(tag + "_stored")
        self.emit("s_waitcnt vmcnt(0)", f"s_branch {self.L('end')}")

    # ---------------------------------------------------------------- kernel
    def kernel(self):
        T = V_T
        self.emit(f"s_load_dwordx16 {sp(S_ARG, 16)}, s[0:1], 0x0",
                  f"s_load_dwordx8 {sp(S_ARG + 16, 8)}, s[0:1], 0x40",
                  f"v_lshrrev_b32_e32 {vp(T)}, 6, {vp(V_TID)}",
                  "s_nop 1",
                  f"v_readfirstlane_b32 {sp(S_WAVE)}, {vp(T)}",
                  "s_waitcnt lgkmcnt(0)",
                  f"s_lshl_b32 {sp(S_M0A)}, {sp(S_WAVE)}, 12",
                  f"s_lshl_b32 {sp(S_M0H)}, {sp(S_WAVE)}, 11",
                  # XCD-aware work: XCD x (workgroups are dealt round robin) takes
                  # whole tiles x per_xcd .. x per_xcd + per_xcd - 1 (below n_whole),
                  # then half pieces x per_xcd_h .. (piece p: tile n_whole + p / 2,
                  # column half p % 2)
                  f"s_and_b32 {sp(S_X)}, s2, 7",
                  f"s_lshr_b32 {sp(S_Y)}, s2, 3",
                  f"s_mov_b32 {sp(S_HALF)}, -1",
                  f"s_cmp_lt_u32 {sp(S_Y)}, {sp(A_PERXCD)}",
                  f"s_cbranch_scc0 {self.L('half_item')}",
                  f"s_mul_i32 {sp(S_ITEM)}, {sp(S_X)}, {sp(A_PERXCD)}",
                  f"s_add_u32 {sp(S_ITEM)}, {sp(S_ITEM)}, {sp(S_Y)}",
                  f"s_cmp_ge_u32 {sp(S_ITEM)}, {sp(A_NWHOLE)}",
                  f"s_cbranch_scc1 {self.L('end')}",
                  f"s_branch {self.L('item_ok')}",
                  self.L("half_item") + ":",
                  f"s_sub_u32 {sp(S_Y)}, {sp(S_Y)}, {sp(A_PERXCD)}",
                  f"s_mul_i32 {sp(S_Z)}, {sp(S_X)}, {sp(A_PERXCDH)}",
                  f"s_add_u32 {sp(S_Z)}, {sp(S_Z)}, {sp(S_Y)}",
                  f"s_cmp_ge_u32 {sp(S_Z)}, {sp(A_NHALF)}",
                  f"s_cbranch_scc1 {self.L('end')}",
                  f"s_and_b32 {sp(S_HALF)}, {sp(S_Z)}, 1",
                  f"s_lshr_b32 {sp(S_Z)}, {sp(S_Z)}, 1",
                  f"s_add_u32 {sp(S_ITEM)}, {sp(A_NWHOLE)}, {sp(S_Z)}",
                  self.L("item_ok") + ":")
        self.decode_tile()
        # A side: rows 256 ti .. (records: the rows that exist, at most 256);
        # W side: rows 256 tj (+ 128 for the second half) .., 256 or 128 of them
        self.emit(f"s_lshl_b32 {sp(S_X)}, {sp(S_TI)}, 8",
                  f"s_mul_hi_u32 {sp(S_Y)}, {sp(S_X)}, {sp(A_LD)}",
                  f"s_mul_i32 {sp(S_Z)}, {sp(S_X)}, {sp(A_LD)}",
                  f"s_add_u32 {sp(S_RA)}, {sp(A_A)}, {sp(S_Z)}",
                  f"s_addc_u32 {sp(S_RA + 1)}, {sp(A_A + 1)}, {sp(S_Y)}",
                  f"s_sub_i32 {sp(S_T)}, {sp(A_N)}, {sp(S_X)}",
                  f"s_min_i32 {sp(S_T)}, {sp(S_T)}, 256",
                  f"s_sub_i32 {sp(S_T)}, {sp(S_T)}, 1",
                  f"s_mul_i32 {sp(S_RECA)}, {sp(S_T)}, {sp(A_LD)}",
                  f"s_add_u32 {sp(S_RECA)}, {sp(S_RECA)}, 64",
                  f"s_lshl_b32 {sp(S_X)}, {sp(S_TJ)}, 8",
                  f"s_max_i32 {sp(S_Y)}, {sp(S_HALF)}, 0",
                  f"s_lshl_b32 {sp(S_Y)}, {sp(S_Y)}, 7",
                  f"s_add_u32 {sp(S_X)}, {sp(S_X)}, {sp(S_Y)}",
                  f"s_mul_hi_u32 {sp(S_Y)}, {sp(S_X)}, {sp(A_LD)}",
                  f"s_mul_i32 {sp(S_Z)}, {sp(S_X)}, {sp(A_LD)}",
                  f"s_add_u32 {sp(S_RB)}, {sp(A_W)}, {sp(S_Z)}",
                  f"s_addc_u32 {sp(S_RB + 1)}, {sp(A_W + 1)}, {sp(S_Y)}",
                  f"s_movk_i32 {sp(S_T)}, 127",
                  f"s_cmp_lt_i32 {sp(S_HALF)}, 0",
                  f"s_cselect_b32 {sp(S_T)}, 255, {sp(S_T)}",
                  f"s_mul_i32 {sp(S_RECB)}, {sp(S_T)}, {sp(A_LD)}",
                  f"s_add_u32 {sp(S_RECB)}, {sp(S_RECB)}, 64",
                  f"s_mov_b32 {sp(S_RA + 3)}, 0x20000",
                  f"s_mov_b32 {sp(S_RB + 3)}, 0x20000",
                  f"s_mov_b32 {sp(S_SLD)}, 0",
                  f"s_mov_b32 {sp(S_STEP)}, 0",
                  f"s_add_u32 {sp(S_BUDGET)}, {sp(A_STEPS)}, 4")
        self.lane_constants()
        for i in range(N_AGPR):
            self.emit(f"v_accvgpr_write_b32 {ap(i)}, 0")
        self.emit(f"s_cmp_lt_i32 {sp(S_HALF)}, 0", f"s_cbranch_scc0 {self.L('half_tile')}")
        self.loop(4, "w")
        self.epilogue(4, "w")
        self.label("half_tile")
        self.loop(2, "h")
        self.epilogue(2, "h")
        self.label("end")
        self.emit("s_waitcnt vmcnt(0)", "s_endpgm")

    def descriptor(self):
        return f"""
\t.section .rodata,"a",@progbits
\t.p2align 6, 0x0
\t.amdhsa_kernel {self.name}
\t\t.amdhsa_group_segment_fixed_size {LDS_BYTES}
\t\t.amdhsa_private_segment_fixed_size 0
\t\t.amdhsa_kernarg_size {ARGS_BYTES}
\t\t.amdhsa_user_sgpr_count 2
\t\t.amdhsa_user_sgpr_kernarg_segment_ptr 1
\t\t.amdhsa_system_sgpr_workgroup_id_x 1
\t\t.amdhsa_system_vgpr_workitem_id 0
\t\t.amdhsa_next_free_vgpr {N_VGPR + N_AGPR}
\t\t.amdhsa_next_free_sgpr {N_SGPR}
\t\t.amdhsa_accum_offset {N_VGPR}
\t\t.amdhsa_reserve_vcc 1
\t\t.amdhsa_float_denorm_mode_32 3
\t\t.amdhsa_float_denorm_mode_16_64 3
\t\t.amdhsa_dx10_clamp 1
\t\t.amdhsa_ieee_mode 1
\t.end_amdhsa_kernel
"""

    def metadata(self):
        return f"""  - .agpr_count:     {N_AGPR}
    .args:
      - .offset:         0
        .size:           {ARGS_BYTES}
        .value_kind:     by_value
    .group_segment_fixed_size: {LDS_BYTES}
    .kernarg_segment_align: 8
    .kernarg_segment_size: {ARGS_BYTES}
    .max_flat_workgroup_size: 256
    .name:           {self.name}
    .private_segment_fixed_size: 0
    .sgpr_count:     {N_SGPR + 2}
    .sgpr_spill_count: 0
    .symbol:         {self.name}.kd
    .uniform_work_group_size: 1
    .vgpr_count:     {N_VGPR + N_AGPR}
    .vgpr_spill_count: 0
    .wavefront_size: 64
"""

    def text(self):
        self.kernel()
        head = f"""\t.text
\t.globl {self.name}
\t.p2align 8
\t.type {self.name},@function
{self.name}:
"""
        return head + "\n".join(self.lines) + "\n" + self.descriptor()


def generate():
    gens = [Gen(False), Gen(True)]
    out = ['\t.amdgcn_target "amdgcn-amd-amdhsa--gfx950"', "\t.amdhsa_code_object_version 5"]
    for g in gens:
        out.append(g.text())
    out.append("\t.amdgpu_metadata\n---\namdhsa.kernels:")
    for g in gens:
        out.append(g.metadata().rstrip("\n"))
    out.append("amdhsa.target:   amdgcn-amd-amdhsa--gfx950\namdhsa.version:\n  - 1\n  - 2\n...\n\t.end_amdgpu_metadata")
    return "\n".join(out) + "\n"


if __name__ == "__main__":
    print(generate())
