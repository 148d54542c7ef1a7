"""Generates gram_fast.s: the gfx950 assembly of the warmup-statistics Gram
kernel for widths that are multiples of 256 (Sec. 3.2: the closed-form
modulation needs the sums X^T X and X^T R over the warmup rows).

G += X^T X on the lower block triangle of 256 x 256 tiles and C += X^T R on
all of them; X [rows, d_in] and R [rows, d_out] are bf16, row-major, and the
contraction runs over the rows, so both MFMA operands come from the LDS
transpose read. One workgroup of 4 waves (one per SIMD) per output tile; wave
(wr, wc) owns the 128 x 128 quarter at rows 128 wr, columns 128 wc, as 4 x 4
accumulation blocks of 32 x 32 fp32 in its 256 accumulation registers, so each
operand read from LDS feeds four matrix instructions.

Rows go HBM -> LDS by buffer loads straight into LDS, 32 rows a stage, in a
ring of four stages (three ahead). A stage holds the tile's 256 X columns
(region A) and its 256 X or R columns (region B), each as two 128-column halves
of 32 rows x 256 bytes with the 16-byte chunks XOR-swizzled by row, the layout
the transpose reads need. Rows past the last one read as zero through the
buffer records, so a ragged last stage needs no branch.

Per stage: phase 0 issues the 16 MFMAs of the first 16-row slice, the reads of
the second slice and the loads of stage s + 3; phase 1 issues 4 MFMAs of the
second slice, waits for stage s + 1 (its own loads, then the barrier that makes
everyone's visible and frees the buffer stage s + 3 will use next time), then
the other 12 MFMAs with the reads of stage s + 1's first slice.

The work list is the C++ Gram kernel's panel-group order (four row panels at a
time: the group's G tiles column by column, then its C tiles), cut into one
contiguous range per XCD, so the workgroups resident on an XCD stream few
distinct panels through its L2. The epilogue adds each block to G or C with
one read-modify-write per element (no atomics: every element is written by
one workgroup, in a fixed order). Tiles that would leave a round of the chip
mostly idle (the last round, or all of them when there are fewer tiles than
compute units) are cut into 2^k row pieces: piece 0 adds into G or C, the
others store their sums to workspace slots that a fixed-order add applies
after the launch.

Run as a script it prints the assembly; build.py assembles it.
"""

KNAME = "ispa_gram_fast"
ARGS_BYTES = 96

# kernel arguments (byte offsets)
ARG_X, ARG_R, ARG_G, ARG_C = 0, 8, 16, 24
ARG_ROWS, ARG_LDX, ARG_LDR, ARG_LDG, ARG_LDC = 32, 36, 40, 44, 48
ARG_TIN, ARG_TOUT, ARG_NT, ARG_PERXCD, ARG_STEPS = 52, 56, 60, 64, 68
ARG_NWHOLE, ARG_PERXCDH, ARG_SPLIT, ARG_LOGS, ARG_WS = 72, 76, 80, 84, 88

S_ARG = 8                       # s[8:31]


def arg(off):
    return S_ARG + off // 4


A_X, A_R, A_G, A_C = arg(ARG_X), arg(ARG_R), arg(ARG_G), arg(ARG_C)
A_ROWS, A_LDX, A_LDR, A_LDG, A_LDC = (arg(o) for o in (ARG_ROWS, ARG_LDX, ARG_LDR, ARG_LDG, ARG_LDC))
A_TIN, A_TOUT, A_NT, A_PERXCD, A_STEPS = (arg(o) for o in (ARG_TIN, ARG_TOUT, ARG_NT, ARG_PERXCD, ARG_STEPS))
A_NWHOLE, A_PERXCDH, A_SPLIT, A_LOGS, A_WS = (arg(o) for o in (ARG_NWHOLE, ARG_PERXCDH, ARG_SPLIT, ARG_LOGS, ARG_WS))

# SGPRs
S_RA = (32, 36)                 # resources of region A halves 0 / 1
S_RB = (40, 44)                 # region B halves 0 / 1
S_PA, S_PB = 48, 50             # 64-bit: the sides' column bases (first row)
S_OA, S_OB = 52, 54             # 64-bit: row offsets (bytes) of the next stage to load
S_MA, S_MB = 56, 57             # remaining bytes from the next stage's row on (records)
S_LDB = 58                      # row bytes of side B (X or R)
S_WAVE, S_W2K = 59, 60          # wave, wave * 2048
S_ITEM, S_TI, S_TJ, S_ISG = 61, 62, 63, 64
S_K, S_R0, S_GM, S_NG, S_N, S_T = 65, 66, 67, 68, 69, 70
S_STEP, S_BUDGET = 71, 72
S_PIECE, S_NSTEPS, S_RB0, S_RE = 96, 97, 98, 99   # piece (-1 whole, 0 ..), its stages, first / end row
S_X, S_Y, S_Z = 73, 74, 75
S_OUT = 76                      # 4: output resource
S_EO = 80                       # 16: epilogue row offsets (bytes) of accumulator element r

# VGPRs
V_TID, V_LANE = 0, 1
V_RA = 2                        # 8: A-side transpose-read addresses, [blk * 2 + h]
V_RB = 10                       # 8: B-side
V_SA = 18                       # 2: staging voffsets, side A, load q
V_SB = 20                       # 2: side B
V_OPS = (24, 56)                # operand sets X / Y: A blocks at +4 b, B blocks at +16 + 4 b
V_T = 88                        # temporaries
N_VGPR = 128
N_AGPR = 256

REGION_B = 65536
STAGE_BYTES = 16384             # one region's share of a stage: two 128-column halves of 32 rows
HALF_BYTES = 8192
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
        self.uid = 0

    def new_uid(self):
        self.uid += 1
        return self.uid

    def emit(self, *ins):
        for i in ins:
            self.lines.append("  " + i if not i.endswith(":") else i)

    # ---------------------------------------------------------------- setup
    def decode_tile(self):
        """S_ITEM -> (S_TI, S_TJ, S_ISG) in panel-group order: row panels four
        at a time; within a group the G tiles of the lower block triangle left
        of and on its diagonal block, column by column, then its C tiles column
        by column."""
        k, r0, gm, ng, n, t = S_K, S_R0, S_GM, S_NG, S_N, S_T
        self.emit(f"s_mov_b32 {sp(k)}, {sp(S_ITEM)}", f"s_mov_b32 {sp(r0)}, 0",
                  ".Lgrp:",
                  f"s_sub_i32 {sp(gm)}, {sp(A_TIN)}, {sp(r0)}",
                  f"s_min_i32 {sp(gm)}, {sp(gm)}, 4",
                  f"s_mul_i32 {sp(ng)}, {sp(r0)}, {sp(gm)}",                # r0 gm
                  f"s_add_i32 {sp(t)}, {sp(gm)}, 1",
                  f"s_mul_i32 {sp(t)}, {sp(t)}, {sp(gm)}",
                  f"s_lshr_b32 {sp(t)}, {sp(t)}, 1",                        # gm (gm + 1) / 2
                  f"s_add_i32 {sp(ng)}, {sp(ng)}, {sp(t)}",                 # G tiles of the group
                  f"s_mul_i32 {sp(n)}, {sp(A_TOUT)}, {sp(gm)}",
                  f"s_add_i32 {sp(n)}, {sp(n)}, {sp(ng)}",
                  f"s_cmp_lt_i32 {sp(k)}, {sp(n)}",
                  "s_cbranch_scc1 .Lgrp_found",
                  f"s_sub_i32 {sp(k)}, {sp(k)}, {sp(n)}",
                  f"s_add_i32 {sp(r0)}, {sp(r0)}, 4",
                  f"s_cmp_lt_i32 {sp(r0)}, {sp(A_TIN)}",
                  "s_cbranch_scc1 .Lgrp",
                  "s_branch .Lend",                                         # past the work list
                  ".Lgrp_found:",
                  f"s_mul_i32 {sp(t)}, {sp(r0)}, {sp(gm)}",
                  f"s_cmp_lt_i32 {sp(k)}, {sp(t)}",
                  "s_cbranch_scc0 .Ldiag",
                  # a full column left of the diagonal block: tj = k / gm, ti = r0 + k % gm
                  f"s_mov_b32 {sp(S_ISG)}, 1",
                  ".Lcolq:")
        self.divmod_gm(".Lcolq", ".Lcolq_done")
        self.emit(".Lcolq_done:",
                  f"s_add_i32 {sp(S_TI)}, {sp(r0)}, {sp(k)}",
                  "s_branch .Ltile_ok",
                  ".Ldiag:",
                  f"s_cmp_lt_i32 {sp(k)}, {sp(ng)}",
                  "s_cbranch_scc0 .Lctile",
                  # the diagonal block's lower triangle: column tj holds rows tj .. r0 + gm - 1
                  f"s_sub_i32 {sp(k)}, {sp(k)}, {sp(t)}",
                  f"s_mov_b32 {sp(S_TJ)}, {sp(r0)}",
                  f"s_mov_b32 {sp(S_ISG)}, 1",
                  ".Ldiag_col:",
                  f"s_add_i32 {sp(t)}, {sp(r0)}, {sp(gm)}",
                  f"s_sub_i32 {sp(t)}, {sp(t)}, {sp(S_TJ)}",
                  f"s_cmp_lt_i32 {sp(k)}, {sp(t)}",
                  "s_cbranch_scc1 .Ldiag_done",
                  f"s_sub_i32 {sp(k)}, {sp(k)}, {sp(t)}",
                  f"s_add_i32 {sp(S_TJ)}, {sp(S_TJ)}, 1",
                  "s_branch .Ldiag_col",
                  ".Ldiag_done:",
                  f"s_add_i32 {sp(S_TI)}, {sp(S_TJ)}, {sp(k)}",
                  "s_branch .Ltile_ok",
                  ".Lctile:",
                  f"s_sub_i32 {sp(k)}, {sp(k)}, {sp(ng)}",
                  f"s_mov_b32 {sp(S_ISG)}, 0",
                  ".Lcq:")
        self.divmod_gm(".Lcq", ".Lcq_done")
        self.emit(".Lcq_done:",
                  f"s_add_i32 {sp(S_TI)}, {sp(r0)}, {sp(k)}",
                  ".Ltile_ok:")

    def divmod_gm(self, top, done):
        """S_TJ = S_K / S_GM, S_K = S_K % S_GM by subtraction (S_GM <= 4)."""
        u = self.new_uid()
        self.emit(f"s_mov_b32 {sp(S_TJ)}, 0",
                  f".Ldm{u}:",
                  f"s_cmp_lt_i32 {sp(S_K)}, {sp(S_GM)}",
                  f"s_cbranch_scc1 {done}",
                  f"s_sub_i32 {sp(S_K)}, {sp(S_K)}, {sp(S_GM)}",
                  f"s_add_i32 {sp(S_TJ)}, {sp(S_TJ)}, 1",
                  f"s_branch .Ldm{u}")
        del top

    def lane_constants(self):
        T = V_T
        self.emit(f"v_and_b32_e32 {vp(V_LANE)}, 63, {vp(V_TID)}")
        # transpose-read addresses (one 128-column half of 32 rows x 256 bytes):
        # g = lane >> 4, sl = lane & 15; for block b of the half and row half h:
        # row = 8 (g >> 1) + 4 h + (sl >> 2), chunk = 4 b + 2 (g & 1) + ((sl & 3) >> 1),
        # address = row * 256 + ((chunk ^ swz(row)) << 4) + 8 (sl & 1),
        # swz(row) = 4 (row & 3) ^ 2 ((row >> 2) & 1)
        self.emit(f"v_lshrrev_b32_e32 {vp(T)}, 4, {vp(V_LANE)}",            # g
                  f"v_and_b32_e32 {vp(T + 1)}, 15, {vp(V_LANE)}",           # sl
                  f"v_lshrrev_b32_e32 {vp(T + 2)}, 1, {vp(T)}",
                  f"v_lshlrev_b32_e32 {vp(T + 2)}, 3, {vp(T + 2)}",         # 8 (g >> 1)
                  f"v_lshrrev_b32_e32 {vp(T + 3)}, 2, {vp(T + 1)}",         # sl >> 2
                  f"v_add_u32_e32 {vp(T + 2)}, {vp(T + 2)}, {vp(T + 3)}",   # row for h = 0
                  f"v_and_b32_e32 {vp(T + 4)}, 1, {vp(T)}",
                  f"v_lshlrev_b32_e32 {vp(T + 4)}, 1, {vp(T + 4)}",         # 2 (g & 1)
                  f"v_bfe_u32 {vp(T + 5)}, {vp(T + 1)}, 1, 1",              # (sl & 3) >> 1
                  f"v_add_u32_e32 {vp(T + 4)}, {vp(T + 4)}, {vp(T + 5)}",   # chunk for b = 0
                  f"v_and_b32_e32 {vp(T + 6)}, 1, {vp(T + 1)}",
                  f"v_lshlrev_b32_e32 {vp(T + 6)}, 3, {vp(T + 6)}")         # 8 (sl & 1)
        # the wave's halves: A half wr, B half wc (wave = 2 wr + wc)
        self.emit(f"s_lshr_b32 {sp(S_X)}, {sp(S_WAVE)}, 1",
                  f"s_lshl_b32 {sp(S_X)}, {sp(S_X)}, 13",                   # A: wr * 8192
                  f"s_and_b32 {sp(S_Y)}, {sp(S_WAVE)}, 1",
                  f"s_lshl_b32 {sp(S_Y)}, {sp(S_Y)}, 13",
                  f"s_add_u32 {sp(S_Y)}, {sp(S_Y)}, {REGION_B}")            # B: 64K + wc * 8192
        for h in range(2):
            self.emit(f"v_add_u32_e32 {vp(T + 7)}, {4 * h}, {vp(T + 2)}",   # row
                      f"v_and_b32_e32 {vp(T + 8)}, 3, {vp(T + 7)}",
                      f"v_lshlrev_b32_e32 {vp(T + 8)}, 2, {vp(T + 8)}",
                      f"v_bfe_u32 {vp(T + 9)}, {vp(T + 7)}, 2, 1",
                      f"v_lshlrev_b32_e32 {vp(T + 9)}, 1, {vp(T + 9)}",
                      f"v_xor_b32_e32 {vp(T + 8)}, {vp(T + 8)}, {vp(T + 9)}")  # swz(row)
            for b in range(4):
                self.emit(f"v_add_u32_e32 {vp(T + 10)}, {4 * b}, {vp(T + 4)}",
                          f"v_xor_b32_e32 {vp(T + 10)}, {vp(T + 10)}, {vp(T + 8)}",
                          f"v_lshlrev_b32_e32 {vp(T + 10)}, 4, {vp(T + 10)}",
                          f"v_lshl_add_u32 {vp(T + 10)}, {vp(T + 7)}, 8, {vp(T + 10)}",
                          f"v_add_u32_e32 {vp(T + 10)}, {vp(T + 10)}, {vp(T + 6)}",
                          f"v_add_u32_e32 {vp(V_RA + 2 * b + h)}, {sp(S_X)}, {vp(T + 10)}",
                          f"v_add_u32_e32 {vp(V_RB + 2 * b + h)}, {sp(S_Y)}, {vp(T + 10)}")
        # staging: lane l of wave w, load q of a half: row = 8 w + 4 q + (l >> 4),
        # stored chunk p = l & 15 holds global chunk p ^ swz(row), swz(row) =
        # 4 (l >> 4) ^ 2 (q & 1); voffset = row * ld + chunk * 16 - 1024 q (the
        # instruction offset 1024 q applies to the memory and the LDS address)
        self.emit(f"v_lshrrev_b32_e32 {vp(T)}, 4, {vp(V_LANE)}",            # l >> 4
                  f"v_and_b32_e32 {vp(T + 1)}, 15, {vp(V_LANE)}",
                  f"s_lshl_b32 {sp(S_X)}, {sp(S_WAVE)}, 3",
                  f"v_add_u32_e32 {vp(T + 2)}, {sp(S_X)}, {vp(T)}",         # 8 w + (l >> 4)
                  f"v_lshlrev_b32_e32 {vp(T + 3)}, 2, {vp(T)}")             # 4 (l >> 4)
        for q in range(2):
            self.emit(f"v_add_u32_e32 {vp(T + 4)}, {4 * q}, {vp(T + 2)}",   # row
                      f"v_xor_b32_e32 {vp(T + 5)}, {2 * (q & 1)}, {vp(T + 3)}",
                      f"v_xor_b32_e32 {vp(T + 5)}, {vp(T + 5)}, {vp(T + 1)}",
                      f"v_lshlrev_b32_e32 {vp(T + 5)}, 4, {vp(T + 5)}",     # chunk bytes
                      f"v_mul_lo_u32 {vp(T + 6)}, {vp(T + 4)}, {sp(A_LDX)}",
                      f"v_add_u32_e32 {vp(T + 6)}, {vp(T + 6)}, {vp(T + 5)}",
                      f"v_subrev_u32_e32 {vp(V_SA + q)}, {1024 * q}, {vp(T + 6)}",
                      f"v_mul_lo_u32 {vp(T + 6)}, {vp(T + 4)}, {sp(S_LDB)}",
                      f"v_add_u32_e32 {vp(T + 6)}, {vp(T + 6)}, {vp(T + 5)}",
                      f"v_subrev_u32_e32 {vp(V_SB + q)}, {1024 * q}, {vp(T + 6)}")

    # ---------------------------------------------------------------- staging
    def stage_list(self, buf):
        """The direct loads of the next stage (rows S_OA / S_OB on) into ring
        buffer `buf`, and the advance of the side cursors by 32 rows, as an
        instruction list. Past the last row the records are 0 (zero fill)."""
        ins = []
        for side, (res, base, off, rem, ld, vs, region) in enumerate(
                ((S_RA, S_PA, S_OA, S_MA, A_LDX, V_SA, 0), (S_RB, S_PB, S_OB, S_MB, S_LDB, V_SB, REGION_B))):
            for half in range(2):
                r = res[half]
                ins += [f"s_add_u32 {sp(r)}, {sp(base)}, {sp(off)}\n"
                        f"  s_addc_u32 {sp(r + 1)}, {sp(base + 1)}, {sp(off + 1)}"]
                if half:
                    ins += [f"s_add_u32 {sp(r)}, {sp(r)}, 256\n  s_addc_u32 {sp(r + 1)}, {sp(r + 1)}, 0",
                            f"s_sub_i32 {sp(r + 2)}, {sp(rem)}, 256"]
                else:
                    ins += [f"s_mov_b32 {sp(r + 2)}, {sp(rem)}"]
                ins += [f"s_max_i32 {sp(r + 2)}, {sp(r + 2)}, 0"]
                lds = region + buf * STAGE_BYTES + half * HALF_BYTES
                ins += [f"s_add_u32 m0, {sp(S_W2K)}, {lds}\n  s_nop 0"]
                ins += [f"buffer_load_dwordx4 {vp(vs + q)}, {sp(r, 4)}, 0 offen offset:{1024 * q} lds"
                        for q in range(2)]
            ins += [f"s_lshl_b32 {sp(S_Z)}, {sp(ld)}, 5",
                    f"s_add_u32 {sp(off)}, {sp(off)}, {sp(S_Z)}\n  s_addc_u32 {sp(off + 1)}, {sp(off + 1)}, 0",
                    f"s_sub_i32 {sp(rem)}, {sp(rem)}, {sp(S_Z)}"]
        return ins

    # ---------------------------------------------------------------- matrix work
    @staticmethod
    def reads(buf, slice_, ops):
        """The 16 transpose reads of one 16-row slice: A blocks then B blocks."""
        imm = buf * STAGE_BYTES + slice_ * 16 * 256
        out = []
        for b in range(4):
            for h in range(2):
                out.append(f"ds_read_b64_tr_b16 {vp(ops + 4 * b + 2 * h, 2)}, {vp(V_RA + 2 * b + h)} offset:{imm}")
        for b in range(4):
            for h in range(2):
                out.append(f"ds_read_b64_tr_b16 {vp(ops + 16 + 4 * b + 2 * h, 2)}, {vp(V_RB + 2 * b + h)} offset:{imm}")
        return out

    @staticmethod
    def mfmas(ops):
        """acc(ai, bj) += A_ai B_bj over one slice: 16 independent accumulations."""
        out = []
        for ai in range(4):
            for bj in range(4):
                acc = ap(16 * (4 * ai + bj), 16)
                out.append(f"v_mfma_f32_32x32x16_bf16 {acc}, {vp(ops + 4 * ai, 4)}, {vp(ops + 16 + 4 * bj, 4)}, {acc}")
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

    def stage_body(self, B):
        """Stage s in ring buffer B; its first slice's operands are in set X."""
        X, Y = V_OPS
        nb = (B + 1) & 3
        self.emit(f".Lstage{B}:",
                  f"s_sub_i32 {sp(S_BUDGET)}, {sp(S_BUDGET)}, 1",
                  f"s_cmp_lt_i32 {sp(S_BUDGET)}, 0",
                  "s_cbranch_scc1 .Lend",
                  "s_waitcnt lgkmcnt(0)")
        # phase 0: slice 0 | reads of slice 1 (set Y; the MFMAs reading Y last
        # were issued a phase ago) | loads of stage s + 3 into buffer (B + 3) & 3
        other = self.reads(B, 1, Y) + self.stage_list((B + 3) & 3)
        self.interleave(self.mfmas(X), other, start=1)
        # phase 1: slice 1 (set Y) | wait for stage s + 1 | reads of its slice 0 (set X)
        m = self.mfmas(Y)
        self.emit("s_waitcnt lgkmcnt(0)")
        for i in m[:4]:
            self.emit(i)
        # every wave's loads of stage s + 1 have landed (at most the loads of
        # stages s + 2 and s + 3, 16, are outstanding per wave) and every wave is
        # done with stage s - 1's buffer
        self.emit("s_waitcnt vmcnt(16)", "s_barrier")
        self.interleave(m[4:], self.reads(nb, 0, X), start=0)
        self.emit(f"s_add_u32 {sp(S_STEP)}, {sp(S_STEP)}, 1",
                  f"s_cmp_ge_u32 {sp(S_STEP)}, {sp(S_NSTEPS)}",
                  "s_cbranch_scc1 .Ldone")
        if B == 3:
            self.emit("s_branch .Lstage0")

    # ---------------------------------------------------------------- epilogue
    def epilogue(self):
        """out[rows of this wave's quarter][cols] += the accumulators; the
        later row pieces of a split tile write their sums to their workspace
        slots instead (a fixed-order add follows the launch)."""
        T = V_T
        self.label(".Ldone")
        # every MFMA has completed before the accumulation registers are read
        self.emit("s_waitcnt vmcnt(0) lgkmcnt(0)", "s_nop 7", "s_nop 7", "s_nop 7")
        # output: G or C from the tile's first element (row 256 ti, column 256 tj),
        # or workspace slot (tile - n_whole) of 256 x 256 fp32 (row bytes 1024)
        u = self.new_uid()
        self.emit(f"s_cmp_gt_i32 {sp(S_PIECE)}, 0",
                  f"s_cbranch_scc1 .Lout_ws{u}",
                  f"s_cmp_eq_u32 {sp(S_ISG)}, 0",
                  f"s_cbranch_scc1 .Lout_c{u}",
                  f"s_mov_b64 {sp(S_OUT, 2)}, {sp(A_G, 2)}",
                  f"s_mov_b32 {sp(S_Z)}, {sp(A_LDG)}",
                  f"s_branch .Lout_rc{u}",
                  f".Lout_c{u}:",
                  f"s_mov_b64 {sp(S_OUT, 2)}, {sp(A_C, 2)}",
                  f"s_mov_b32 {sp(S_Z)}, {sp(A_LDC)}",
                  f".Lout_rc{u}:",
                  f"s_lshl_b32 {sp(S_X)}, {sp(S_TI)}, 8",
                  f"s_mul_hi_u32 {sp(S_Y)}, {sp(S_X)}, {sp(S_Z)}",
                  f"s_mul_i32 {sp(S_X)}, {sp(S_X)}, {sp(S_Z)}",
                  f"s_add_u32 {sp(S_OUT)}, {sp(S_OUT)}, {sp(S_X)}",
                  f"s_addc_u32 {sp(S_OUT + 1)}, {sp(S_OUT + 1)}, {sp(S_Y)}",
                  f"s_lshl_b32 {sp(S_X)}, {sp(S_TJ)}, 10",                   # 256 tj * 4 bytes
                  f"s_add_u32 {sp(S_OUT)}, {sp(S_OUT)}, {sp(S_X)}",
                  f"s_addc_u32 {sp(S_OUT + 1)}, {sp(S_OUT + 1)}, 0",
                  f"s_branch .Lout_ok{u}",
                  f".Lout_ws{u}:",
                  # slot (piece - 1) * split tiles + (tile - n_whole)
                  f"s_sub_u32 {sp(S_X)}, {sp(A_NT)}, {sp(A_NWHOLE)}",
                  f"s_sub_u32 {sp(S_Y)}, {sp(S_PIECE)}, 1",
                  f"s_mul_i32 {sp(S_X)}, {sp(S_X)}, {sp(S_Y)}",
                  f"s_add_u32 {sp(S_X)}, {sp(S_X)}, {sp(S_ITEM)}",
                  f"s_sub_u32 {sp(S_X)}, {sp(S_X)}, {sp(A_NWHOLE)}",
                  f"s_lshr_b32 {sp(S_Y)}, {sp(S_X)}, 14",
                  f"s_lshl_b32 {sp(S_X)}, {sp(S_X)}, 18",                    # 256 KB per slot
                  f"s_add_u32 {sp(S_OUT)}, {sp(A_WS)}, {sp(S_X)}",
                  f"s_addc_u32 {sp(S_OUT + 1)}, {sp(A_WS + 1)}, {sp(S_Y)}",
                  f"s_movk_i32 {sp(S_Z)}, 0x400",
                  f".Lout_ok{u}:",
                  # the wave's quarter: + 128 wr rows, + 128 wc columns
                  f"s_lshr_b32 {sp(S_X)}, {sp(S_WAVE)}, 1",
                  f"s_lshl_b32 {sp(S_X)}, {sp(S_X)}, 7",
                  f"s_mul_i32 {sp(S_X)}, {sp(S_X)}, {sp(S_Z)}",
                  f"s_and_b32 {sp(S_Y)}, {sp(S_WAVE)}, 1",
                  f"s_lshl_b32 {sp(S_Y)}, {sp(S_Y)}, 9",                     # 128 wc * 4 bytes
                  f"s_add_u32 {sp(S_X)}, {sp(S_X)}, {sp(S_Y)}",
                  f"s_add_u32 {sp(S_OUT)}, {sp(S_OUT)}, {sp(S_X)}",
                  f"s_addc_u32 {sp(S_OUT + 1)}, {sp(S_OUT + 1)}, 0",
                  # records: the quarter's 128 rows
                  f"s_lshl_b32 {sp(S_OUT + 2)}, {sp(S_Z)}, 7",
                  f"s_mov_b32 {sp(S_OUT + 3)}, 0x20000")
        # accumulator element r of lane l: row 8 (r >> 2) + 4 (l >> 5) + (r & 3), column l & 31
        for r in range(16):
            self.emit(f"s_mul_i32 {sp(S_EO + r)}, {sp(S_Z)}, {8 * (r >> 2) + (r & 3)}")
        self.emit(f"v_lshrrev_b32_e32 {vp(T)}, 5, {vp(V_LANE)}",
                  f"v_lshlrev_b32_e32 {vp(T)}, 2, {vp(T)}",                  # 4 (l >> 5)
                  f"v_mul_lo_u32 {vp(T)}, {vp(T)}, {sp(S_Z)}",
                  f"v_and_b32_e32 {vp(T + 1)}, 31, {vp(V_LANE)}",
                  f"v_lshl_add_u32 {vp(T)}, {vp(T + 1)}, 2, {vp(T)}")       # lane's voffset in a block
        # block (ai, bj) adds 32 ai rows and 32 bj columns to the lane's voffset;
        # the read-modify-write is pipelined over two 16-value buffers (the
        # operand registers, free here): the loads of block k + 1 are in flight
        # while block k is added and stored (memory operations retire in order,
        # so vmcnt(16) / vmcnt(32) leave exactly the younger block's loads, or
        # those and the older block's stores, outstanding)
        blocks = [(ai, bj) for ai in range(4) for bj in range(4)]
        VB = (V_OPS[0], V_OPS[0] + 16)
        VO = (V_OPS[1], V_OPS[1] + 1)                                        # voffsets per buffer

        def voff(k):
            ai, bj = blocks[k]
            return [f"s_mul_i32 {sp(S_X)}, {sp(S_Z)}, {32 * ai}",
                    f"s_add_u32 {sp(S_X)}, {sp(S_X)}, {128 * bj}",
                    f"v_add_u32_e32 {vp(VO[k & 1])}, {sp(S_X)}, {vp(T)}"]

        def loads(k):
            return [f"buffer_load_dword {vp(VB[k & 1] + r)}, {vp(VO[k & 1])}, {sp(S_OUT, 4)}, {sp(S_EO + r)} offen"
                    for r in range(16)]

        def stores(k, src):
            return [f"buffer_store_dword {vp(src + r)}, {vp(VO[k & 1])}, {sp(S_OUT, 4)}, {sp(S_EO + r)} offen"
                    for r in range(16)]

        self.emit(f"s_cmp_gt_i32 {sp(S_PIECE)}, 0", f"s_cbranch_scc1 .Lstore_ws{u}")
        self.emit(*voff(0), *loads(0))
        for k in range(16):
            acc = 16 * (4 * blocks[k][0] + blocks[k][1])
            if k + 1 < 16:
                self.emit(*voff(k + 1), *loads(k + 1))
                self.emit("s_waitcnt vmcnt(16)" if k == 0 else "s_waitcnt vmcnt(32)")
            else:
                self.emit("s_waitcnt vmcnt(16)")
            for r in range(16):
                self.emit(f"v_accvgpr_read_b32 {vp(T + 3)}, {ap(acc + r)}",
                          f"v_add_f32_e32 {vp(VB[k & 1] + r)}, {vp(VB[k & 1] + r)}, {vp(T + 3)}")
            self.emit(*stores(k, VB[k & 1]))
        self.emit("s_branch .Lstored")
        # the later row pieces of a split tile: plain stores of the sums
        self.label(f".Lstore_ws{u}")
        for k in range(16):
            acc = 16 * (4 * blocks[k][0] + blocks[k][1])
            self.emit(*voff(k))
            for r in range(16):
                self.emit(f"v_accvgpr_read_b32 {vp(VB[k & 1] + r)}, {ap(acc + r)}")
            self.emit("s_nop 1", *stores(k, VB[k & 1]))
            if k + 1 < 16:
                self.emit("s_waitcnt vmcnt(16)")    # the other buffer's stores have read their data
        self.label(".Lstored")
        self.emit("s_waitcnt vmcnt(0)")

    def label(self, name):
        self.lines.append(name + ":")

    # ---------------------------------------------------------------- kernel
    def kernel(self):
        T = V_T
        self.emit(f"s_load_dwordx16 {sp(S_ARG, 16)}, s[0:1], 0x0",
                  f"s_load_dwordx8 {sp(S_ARG + 16, 8)}, s[0:1], 0x40",
                  f"v_lshrrev_b32_e32 {vp(T)}, 6, {vp(V_TID)}",
                  "s_nop 1",
                  f"v_readfirstlane_b32 {sp(S_WAVE)}, {vp(T)}",
                  "s_waitcnt lgkmcnt(0)",
                  f"s_lshl_b32 {sp(S_W2K)}, {sp(S_WAVE)}, 11",
                  # XCD-aware work: XCD x (workgroups are dealt round robin) takes
                  # whole tiles x per_xcd .. x per_xcd + per_xcd - 1 (tiles below
                  # n_whole), then pieces x per_xcd_h .. of the tiles from n_whole
                  # on, each cut into 2^log_pieces row pieces (piece p: tile
                  # n_whole + p >> log_pieces, rows p mod 2^log_pieces), so that the
                  # last round of a launch is not mostly idle
                  f"s_and_b32 {sp(S_X)}, s2, 7",
                  f"s_lshr_b32 {sp(S_Y)}, s2, 3",
                  f"s_mov_b32 {sp(S_PIECE)}, -1",
                  f"s_cmp_lt_u32 {sp(S_Y)}, {sp(A_PERXCD)}",
                  "s_cbranch_scc0 .Lhalf_item",
                  f"s_mul_i32 {sp(S_ITEM)}, {sp(S_X)}, {sp(A_PERXCD)}",
                  f"s_add_u32 {sp(S_ITEM)}, {sp(S_ITEM)}, {sp(S_Y)}",
                  f"s_cmp_ge_u32 {sp(S_ITEM)}, {sp(A_NWHOLE)}",
                  "s_cbranch_scc1 .Lend",
                  "s_branch .Litem_ok",
                  ".Lhalf_item:",
                  f"s_sub_u32 {sp(S_Y)}, {sp(S_Y)}, {sp(A_PERXCD)}",
                  f"s_mul_i32 {sp(S_Z)}, {sp(S_X)}, {sp(A_PERXCDH)}",
                  f"s_add_u32 {sp(S_Z)}, {sp(S_Z)}, {sp(S_Y)}",                  # piece index p
                  f"s_sub_u32 {sp(S_X)}, {sp(A_NT)}, {sp(A_NWHOLE)}",
                  f"s_lshl_b32 {sp(S_X)}, {sp(S_X)}, {sp(A_LOGS)}",
                  f"s_cmp_ge_u32 {sp(S_Z)}, {sp(S_X)}",
                  "s_cbranch_scc1 .Lend",
                  f"s_lshl_b32 {sp(S_T)}, 1, {sp(A_LOGS)}",
                  f"s_sub_u32 {sp(S_T)}, {sp(S_T)}, 1",
                  f"s_and_b32 {sp(S_PIECE)}, {sp(S_Z)}, {sp(S_T)}",
                  f"s_lshr_b32 {sp(S_Z)}, {sp(S_Z)}, {sp(A_LOGS)}",
                  f"s_add_u32 {sp(S_ITEM)}, {sp(A_NWHOLE)}, {sp(S_Z)}",
                  ".Litem_ok:",
                  # rows of this work item: all, or the split stages of piece q from
                  # stage q split on
                  f"s_mov_b32 {sp(S_RB0)}, 0",
                  f"s_mov_b32 {sp(S_RE)}, {sp(A_ROWS)}",
                  f"s_mov_b32 {sp(S_NSTEPS)}, {sp(A_STEPS)}",
                  f"s_cmp_lt_i32 {sp(S_PIECE)}, 0",
                  "s_cbranch_scc1 .Lrows_ok",
                  f"s_mul_i32 {sp(S_X)}, {sp(A_SPLIT)}, {sp(S_PIECE)}",         # first stage
                  f"s_sub_i32 {sp(S_NSTEPS)}, {sp(A_STEPS)}, {sp(S_X)}",
                  f"s_min_i32 {sp(S_NSTEPS)}, {sp(S_NSTEPS)}, {sp(A_SPLIT)}",
                  f"s_lshl_b32 {sp(S_RB0)}, {sp(S_X)}, 5",
                  f"s_lshl_b32 {sp(S_X)}, {sp(A_SPLIT)}, 5",
                  f"s_add_u32 {sp(S_X)}, {sp(S_X)}, {sp(S_RB0)}",
                  f"s_min_i32 {sp(S_RE)}, {sp(S_RE)}, {sp(S_X)}",
                  ".Lrows_ok:")
        self.decode_tile()
        # side A: X columns 256 ti .. (bytes 512 ti); side B: X (G tile) or R (C tile) columns 256 tj ..
        u = self.new_uid()
        self.emit(f"s_lshl_b32 {sp(S_X)}, {sp(S_TI)}, 9",
                  f"s_add_u32 {sp(S_PA)}, {sp(A_X)}, {sp(S_X)}",
                  f"s_addc_u32 {sp(S_PA + 1)}, {sp(A_X + 1)}, 0",
                  f"s_lshl_b32 {sp(S_Y)}, {sp(S_TJ)}, 9",
                  f"s_cmp_eq_u32 {sp(S_ISG)}, 0",
                  f"s_cbranch_scc1 .Lbside_r{u}",
                  f"s_add_u32 {sp(S_PB)}, {sp(A_X)}, {sp(S_Y)}",
                  f"s_addc_u32 {sp(S_PB + 1)}, {sp(A_X + 1)}, 0",
                  f"s_mov_b32 {sp(S_LDB)}, {sp(A_LDX)}",
                  f"s_branch .Lbside_ok{u}",
                  f".Lbside_r{u}:",
                  f"s_add_u32 {sp(S_PB)}, {sp(A_R)}, {sp(S_Y)}",
                  f"s_addc_u32 {sp(S_PB + 1)}, {sp(A_R + 1)}, 0",
                  f"s_mov_b32 {sp(S_LDB)}, {sp(A_LDR)}",
                  f".Lbside_ok{u}:",
                  # cursors: row 0; records from a stage's row on = the bytes left
                  # in the matrix past the side's column base (rows past the last
                  # one read as zero)
                  f"s_mul_i32 {sp(S_OA)}, {sp(S_RB0)}, {sp(A_LDX)}",
                  f"s_mov_b32 {sp(S_OA + 1)}, 0",
                  f"s_mul_i32 {sp(S_OB)}, {sp(S_RB0)}, {sp(S_LDB)}",
                  f"s_mov_b32 {sp(S_OB + 1)}, 0",
                  f"s_sub_i32 {sp(S_Z)}, {sp(S_RE)}, {sp(S_RB0)}",               # rows of the piece
                  f"s_mul_i32 {sp(S_MA)}, {sp(S_Z)}, {sp(A_LDX)}",
                  f"s_sub_i32 {sp(S_MA)}, {sp(S_MA)}, {sp(S_X)}",
                  f"s_mul_i32 {sp(S_MB)}, {sp(S_Z)}, {sp(S_LDB)}",
                  f"s_sub_i32 {sp(S_MB)}, {sp(S_MB)}, {sp(S_Y)}")
        for r in S_RA + S_RB:
            self.emit(f"s_mov_b32 {sp(r + 3)}, 0x20000")
        self.lane_constants()
        # zero accumulators
        for i in range(N_AGPR):
            self.emit(f"v_accvgpr_write_b32 {ap(i)}, 0")
        # stages 0, 1, 2
        for b in range(3):
            for i in self.stage_list(b):
                self.emit(i)
        self.emit(f"s_mov_b32 {sp(S_STEP)}, 0",
                  f"s_add_u32 {sp(S_BUDGET)}, {sp(S_NSTEPS)}, 4",
                  # stage 0 resident everywhere (the loads of stages 1, 2 may stay in flight)
                  "s_waitcnt vmcnt(16)", "s_barrier")
        for i in self.reads(0, 0, V_OPS[0]):
            self.emit(i)
        for B in range(4):
            self.stage_body(B)
        self.epilogue()
        self.label(".Lend")
        self.emit("s_waitcnt vmcnt(0)", "s_endpgm")

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
\t\t.amdhsa_next_free_vgpr {N_VGPR + N_AGPR}
\t\t.amdhsa_next_free_sgpr 100
\t\t.amdhsa_accum_offset {N_VGPR}
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
    .sgpr_count:     102
    .sgpr_spill_count: 0
    .symbol:         {KNAME}.kd
    .uniform_work_group_size: 1
    .vgpr_count:     {N_VGPR + N_AGPR}
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
    print(generate())
