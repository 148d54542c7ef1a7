// Chunk attention against a KV cache for gfx950 (CDNA4).
//
// Operation (arXiv 2607.00712): softmax attention of the current chunk's
// queries over a set of cached keys (Sec. 2, Eq. 3), where the set is the
// local context (sink prefix + most recent keys, Sec. 3.4 Eq. 7), the history
// (Eq. 8) or both. In the dual-stream form one pass produces both the local
// result and the full result: the online-softmax state after the local keys is
// exactly (O_loc, LSE_loc) of Eq. 9, and continuing the same state over the
// history keys gives the LSE fusion of Eq. 11-12 without a second pass.
//
// Work decomposition
//   workgroup = 8 waves (two per SIMD) = 256 queries of one head; each wave
//   owns 32 queries, and every K / V tile is staged once for all 256.
//   Keys are visited in tiles of 64 rows. Only tiles that intersect the key set
//   are visited; the tile at the end of each contiguous range is masked
//   element-wise.
// Staging: K and V tiles go straight from HBM to LDS with buffer loads
//   (buffer_load_dwordx4 ... lds), double buffered, one barrier per tile. The
//   buffer descriptor of a tile starts at its first key and covers only its
//   valid rows, so rows past the end of a range read as zero in hardware. A
//   direct load writes 64 consecutive 16-byte slots per wave, so LDS rows are
//   unpadded and the 16-byte chunk index is XOR-swizzled with the row
//   (slot = chunk ^ row) to keep the MFMA operand reads and the transpose reads
//   free of bank conflicts.
//
// Per tile and wave (bf16 MFMA 32x32x16, fp32 accumulation), in two halves of
// 32 keys, each a complete online-softmax step:
//   S^T[32 keys x 32 q] = K_half . Q^T   -- A = K rows from LDS, B = Q^T in VGPRs.
//     The accumulator layout gives each lane the scores of ONE query (lane%32)
//     for 32 keys; the other 32 keys of that query sit in lane^32. Row max
//     needs one cross-lane exchange; row sums stay per lane until the end.
//   O^T[D x 32 q] += V_tile^T . P^T   -- B = P^T straight from the score
//     registers (converted to bf16). Within each 16-key slice the score
//     registers hold keys {4h..4h+3, 8+4h..8+4h+3} for lane half h, so the
//     contraction index is permuted; the V^T operand is read with the same
//     permutation by two LDS transpose reads (ds_read_b64_tr_b16), which fetch
//     4 consecutive keys of one column per lane from row-major V.
//   The output accumulator is O^T, so the per-query rescale factor of the
//   online softmax is a per-lane scalar.
//
// Softmax uses exp2 with the logit scale folded into one FMA:
//   p = 2^(s * c - m * c), c = scale * log2(e); LSE = m * scale + ln(l),
// where the reference m trails the running max by at most 8 (log2 units).
//
// Workgroups are remapped so that the 8 XCDs (dispatched round-robin) each own
// a contiguous run of (head, query tile) work items: tiles of one head share
// the K/V stream through one XCD's L2.
#include <stdlib.h>

#include "ispa_internal.h"

#include <limits.h>
#include <math.h>

namespace ispa {
namespace {

constexpr int kWaves = 8;
constexpr int kThreads = kWaves * 64;
constexpr int kBqWave = 32;
constexpr int kBq = kWaves * kBqWave;  // queries per workgroup
static_assert(kBq == kAttnBq, "work item size");
constexpr int kBk = 64;                // keys per tile
constexpr int kXcds = 8;
constexpr float kLazyLog2 = 8.f;       // rescale threshold of the softmax reference
constexpr int kSplitMinTiles = 384;    // automatic split only from this many key tiles per item
constexpr int kSplitFillPct = 85;      // automatic split only below this fill of the last round

template <int D>
struct Cfg {
  static constexpr int rowBytes = D * 2;                     // unpadded LDS row
  static constexpr int chunksPerRow = D / 8;                 // 16-byte chunks
  static constexpr int swz = chunksPerRow - 1;               // XOR mask
  static constexpr int tileBytes = kBk * rowBytes;           // one K or V tile
  static constexpr int loadsPerThread = kBk * chunksPerRow / kThreads;
  static constexpr int kSlices = D / 16;                     // QK^T k-steps
  static constexpr int dBlocks = D / 32;                     // O^T row blocks
  static_assert(kBk * chunksPerRow % kThreads == 0, "tile load split");
};

// XOR swizzles of the 16-byte chunk index, per tile and row.
// K is read as MFMA A operands: 16 lanes read 16 consecutive rows at the same
// logical chunk, so chunk ^ (row mod 16) spreads them over all banks.
// V is read with transpose reads: 16 lanes read 4 consecutive rows x 2 adjacent
// chunks, and the two 16-lane groups that share a lane half read the next two
// chunks of the same rows; chunk ^ (4 * (row mod 4)) gives those 32 lanes 16
// distinct chunk positions, and the extra ^2 for rows 4..7 (mod 8) separates
// the other lane half.
template <int D>
__device__ __forceinline__ int swz_k(int row) { return row & Cfg<D>::swz; }
template <int D>
__device__ __forceinline__ int swz_v(int row) {
  return D == 128 ? ((4 * (row & 3)) ^ (2 * ((row >> 2) & 1))) : (row & Cfg<D>::swz);
}
// byte offset of logical chunk `c` of row `row` for a given swizzle value
template <int D>
__device__ __forceinline__ int chunk_off(int row, int c, int sw) {
  return row * Cfg<D>::rowBytes + ((c ^ sw) << 4);
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int nbytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, nbytes, 0x00020000);
}

__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// V^T operands come from LDS transpose reads issued as inline asm and completed
// by explicit waits tied to their results. Through the builtin the compiler
// cannot tell these reads from reads of the buffer the direct loads are filling,
// and would wait for those loads (vmcnt 0) before every slice. LDS operations
// complete in order, so a wait for "at most n outstanding" retires exactly the
// reads issued before the last n, and the compiler's own lgkmcnt waits, which
// do not count these reads, only become more conservative.
__device__ __forceinline__ uint32_t lds_addr(const char* p) {
  return (uint32_t)(uintptr_t)(ISPA_LDS const char*)p;
}

// The 2 x NB transpose reads of one 16-key slice; IMM is the compile-time byte
// offset of the slice (buffer, V tile, slice rows) from the per-lane addresses.
template <int NB, int IMM>
__device__ __forceinline__ void tr_issue(const uint32_t (&addr)[2][NB], u32x2 (&r)[2][NB]) {
#pragma unroll
  for (int db = 0; db < NB; ++db) {
    asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(r[0][db]) : "v"(addr[0][db]), "i"(IMM));
    asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(r[1][db]) : "v"(addr[1][db]), "i"(IMM));
  }
}

// Wait until at most N LDS operations are outstanding, then hand out the
// slice's operands.
template <int N, int NB>
__device__ __forceinline__ void tr_wait(u32x2 (&r)[2][NB], bf16x8* out) {
  if constexpr (NB == 4) {
    asm volatile("s_waitcnt lgkmcnt(%8)"
                 : "+v"(r[0][0]), "+v"(r[1][0]), "+v"(r[0][1]), "+v"(r[1][1]), "+v"(r[0][2]), "+v"(r[1][2]),
                   "+v"(r[0][3]), "+v"(r[1][3])
                 : "i"(N));
  } else {
    asm volatile("s_waitcnt lgkmcnt(%4)" : "+v"(r[0][0]), "+v"(r[1][0]), "+v"(r[0][1]), "+v"(r[1][1]) : "i"(N));
  }
#pragma unroll
  for (int db = 0; db < NB; ++db) {
    const u32x4 w{r[0][db][0], r[0][db][1], r[1][db][0], r[1][db][1]};
    out[db] = __builtin_bit_cast(bf16x8, w);
  }
}

// The kSlices K operands (A of S^T = K Q^T) of one half; IMM is the
// compile-time byte offset of the half (buffer, half rows). `dep` is a value
// computed from the previous half's scores: taking it as an input orders the
// reads after the MFMAs that consumed the previous contents of r.
template <int NS, int IMM>
__device__ __forceinline__ void k_issue(const uint32_t (&addr)[NS], u32x4 (&r)[NS], float dep) {
#pragma unroll
  for (int kk = 0; kk < NS; ++kk)
    asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(r[kk]) : "v"(addr[kk]), "i"(IMM), "v"(dep));
}
// Wait until K operand `r` (issued N reads before the last one) has arrived.
template <int N>
__device__ __forceinline__ void k_wait_one(u32x4& r) {
  static_assert(N >= 0 && N <= 15, "lgkmcnt range");
  asm volatile("s_waitcnt lgkmcnt(%1)" : "+v"(r) : "i"(N));
}
// S^T += K . Q^T over the slices KK.. of a half, each MFMA after its own wait.
template <int NS, int KK = 0>
__device__ __forceinline__ void qk_chain(u32x4 (&kr)[NS], const bf16x8 (&qf)[NS], f32x16& sc) {
  if constexpr (KK < NS) {
    k_wait_one<NS - 1 - KK>(kr[KK]);
    sc = mfma32(__builtin_bit_cast(bf16x8, kr[KK]), qf[KK], sc);
    // keep the next wait behind this MFMA (only VALU / SALU work may move across)
    __builtin_amdgcn_sched_barrier(0x6);
    qk_chain<NS, KK + 1>(kr, qf, sc);
  }
}
template <int N>
__device__ __forceinline__ void k_wait(u32x4 (&r)[8]) {
  static_assert(N >= 0 && N <= 15, "lgkmcnt range");
  asm volatile("s_waitcnt lgkmcnt(%8)"
               : "+v"(r[0]), "+v"(r[1]), "+v"(r[2]), "+v"(r[3]), "+v"(r[4]), "+v"(r[5]), "+v"(r[6]), "+v"(r[7])
               : "i"(N));
}
template <int N>
__device__ __forceinline__ void k_wait(u32x4 (&r)[4]) {
  static_assert(N >= 0 && N <= 15, "lgkmcnt range");
  asm volatile("s_waitcnt lgkmcnt(%4)" : "+v"(r[0]), "+v"(r[1]), "+v"(r[2]), "+v"(r[3]) : "i"(N));
}

// Lane-pair (l, l ^ 32) exchange with v_permlane32_swap: it swaps the upper 32
// lanes of its first operand with the lower 32 lanes of its second, so with
// A = B = x in two registers it leaves A = [x_lo, x_lo] and B = [x_hi, x_hi].
// Written as inline asm with two in/out operands: the builtin's second result
// was observed to be read back from the first operand's register.
__device__ __forceinline__ void pair_halves(float x, float& lo, float& hi) {
  lo = x;
  hi = x;
  asm volatile("s_nop 1\n\tv_permlane32_swap_b32 %0, %1\n\ts_nop 1" : "+v"(lo), "+v"(hi));
}
__device__ __forceinline__ float l_run_total(float x) {
  float lo, hi;
  pair_halves(x, lo, hi);
  return lo + hi;
}
// Maxima of finite-or-minus-infinity scores as v_maximum3 / v_maximum (fmaxf
// would first quiet possible signalling NaNs with an extra instruction per
// operand; scores are never NaN). They stay compiler-visible instructions:
// the scores are MFMA results, and only the compiler inserts the wait states
// that a VALU read of an MFMA destination needs.
__device__ __forceinline__ float max3(float a, float b, float c) {
  return __builtin_elementwise_maximum(__builtin_elementwise_maximum(a, b), c);
}
__device__ __forceinline__ float max2(float a, float b) { return __builtin_elementwise_maximum(a, b); }
__device__ __forceinline__ float pair_max(float x) {
  float lo, hi;
  pair_halves(x, lo, hi);
  return max2(lo, hi);
}

// The flattened range list, held in registers for the key loop: range i
// covers keys [b_i, e_i) and starts at tile tb_i (tb_i = INT_MAX for an absent
// range). A scalar load inside the loop would also count in lgkmcnt and, unlike
// LDS reads, complete out of order, which the counted LDS waits cannot allow.
struct TileMap {
  int64_t b0, b1, b2, e0, e1, e2;
  int tb1, tb2;
};
// Tile t: first key and number of valid keys.
__device__ __forceinline__ void tile_of(const TileMap& m, int t, int64_t& key0, int& nvalid) {
  // selects of values, not of member lvalues (those would select addresses
  // and keep the map in memory)
  const int64_t b0 = m.b0, b1 = m.b1, b2 = m.b2, e0 = m.e0, e1 = m.e1, e2 = m.e2;
  const int tb1 = m.tb1, tb2 = m.tb2;
  const bool in2 = t >= tb2;
  const bool in1 = !in2 && t >= tb1;
  const int64_t begin = in2 ? b2 : (in1 ? b1 : b0);
  const int64_t end = in2 ? e2 : (in1 ? e1 : e0);
  const int first = in2 ? tb2 : (in1 ? tb1 : 0);
  key0 = begin + (int64_t)(t - first) * kBk;
  const int64_t left = end - key0;
  nvalid = left < kBk ? (int)left : kBk;
}

// Direct HBM -> LDS loads of one K tile and one V tile (kBk rows starting at
// element offset `base`, `nv` of them valid) into dst = [K tile | V tile].
// (A plain function: the host compilation pass drops a kernel whose lambdas
// use the LDS-load builtin.)
template <int D>
__device__ __forceinline__ void stage_tile(const AttnArgs& a, int64_t base, int nv, char* dst,
                                           int voffk, int voffv, int wave) {
  using C = Cfg<D>;
  const int nbytes = (int)(((int64_t)(nv - 1) * a.ld + D) * 2);
  const __amdgpu_buffer_rsrc_t rk = make_rsrc(a.k + base, nbytes);
  const __amdgpu_buffer_rsrc_t rv = make_rsrc(a.v + base, nbytes);
  // load q covers the rows of load 0 plus q * (kThreads / chunksPerRow), with
  // the same swizzles (they depend on the row mod 16)
  const int qstride = (int)((kThreads / C::chunksPerRow) * a.ld * 2);
#pragma unroll
  for (int q = 0; q < C::loadsPerThread; ++q) {
    const int wslot = (q * kWaves + wave) * 64 * 16;  // wave-uniform LDS destination
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, (ISPA_LDS void*)(dst + wslot), 16, voffk + q * qstride, 0, 0, 0);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, (ISPA_LDS void*)(dst + C::tileBytes + wslot), 16,
                                             voffv + q * qstride, 0, 0, 0);
  }
}

// Per-wave state of the online softmax and the per-lane constants of the loop.
template <int D>
struct Wave {
  using C = Cfg<D>;
  f32x16 acc[C::dBlocks];      // O^T, one 32 x 32 block per 32 head dims
  float m_run;                 // softmax reference (raw score units) of this lane's query
  float lazy;                  // kLazyLog2 in raw score units
  float l_run;                 // running sum of p (this lane's half of the keys), for the LSE
  float lr_run;                // running sum of the bf16-rounded p, the normaliser of O
  bf16x8 qf[C::kSlices];       // Q^T operand
  u32x4 kr[C::kSlices];        // K operands of the current half
  uint32_t koff[C::kSlices];   // K operand LDS addresses (buffer 0, half 0)
  uint32_t vaddr[2][C::dBlocks];  // V transpose-read LDS addresses (buffer 0, slice 0)
  int voffk, voffv;            // direct-load offsets of a thread's first load
};

struct Loop {
  TileMap map;
  int n_tiles, n_tiles_local, hoff, wave, hh;
  bool dual;
};

// Writes the normalised output and LSE of this lane's query, either to the
// launch's output rows (slot < 0) or to partial slot `slot` (part `which`:
// 0 end state, 1 local set) of the split.
template <int D>
__device__ __forceinline__ void write_state(const AttnArgs& a, Wave<D>& w, const Loop& L, int qloc, int qrow,
                                            int head, float* out, float* lse, int slot, int which) {
  using C = Cfg<D>;
  const float l_tot = l_run_total(w.l_run);
  const float inv = 1.0f / l_run_total(w.lr_run);
  if (qrow >= a.n_q) return;
  float* op;
  float* lp;
  if (slot < 0) {
    op = out + (int64_t)qrow * a.ld + L.hoff + 4 * L.hh;
    lp = lse != nullptr ? lse + (int64_t)head * a.n_q + qrow : nullptr;
  } else {
    const int64_t base = ((int64_t)slot * 2 + which) * kBq;
    op = a.split.part_o + (base + qloc) * D + 4 * L.hh;
    lp = a.split.part_lse + base + qloc;
  }
#pragma unroll
  for (int db = 0; db < C::dBlocks; ++db) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f32x4 o;
      o[0] = w.acc[db][4 * i + 0] * inv;
      o[1] = w.acc[db][4 * i + 1] * inv;
      o[2] = w.acc[db][4 * i + 2] * inv;
      o[3] = w.acc[db][4 * i + 3] * inv;
      *(f32x4*)(op + 32 * db + 8 * i) = o;
    }
  }
  if (lp != nullptr && L.hh == 0) *lp = w.m_run * a.scale + logf(l_tot);
}

// One 32-key online-softmax step: keys 32B .. 32B+31 of the tile in LDS buffer BUF.
template <int D, int BUF, int B>
__device__ __forceinline__ void half_step(const AttnArgs& a, Wave<D>& w, const Loop& L, const char* smem, int nv) {
  using C = Cfg<D>;
  constexpr int vBase = BUF * 2 * C::tileBytes + C::tileBytes;
  // S^T = K . Q^T (rows 32B + ql share the swizzle of row ql); the K operands
  // of this half are in registers
  // (each MFMA waits only for its own K operand: the reads of this half are
  // the only LDS operations in flight and complete in issue order)
  f32x16 sc = f32x16{};
  qk_chain<C::kSlices>(w.kr, w.qf, sc);
  // V^T operands of this half's two 16-key slices, in flight during the softmax
  u32x2 v0[2][C::dBlocks], v1[2][C::dBlocks];
  tr_issue<C::dBlocks, vBase + 16 * (2 * B) * C::rowBytes>(w.vaddr, v0);
  tr_issue<C::dBlocks, vBase + 16 * (2 * B + 1) * C::rowBytes>(w.vaddr, v1);
  // keys past the end of a range (only in the last tile of each range)
  if (nv < 32 * (B + 1)) {
    // register r holds key 32B + 4 hh + 8 (r / 4) + r % 4 of the tile (compared
    // as a compile-time offset against one limit, so that no per-register key
    // indices stay live across the loop)
    const int lim = nv - 32 * B - 4 * L.hh;
#pragma unroll
    for (int r = 0; r < 16; ++r)
      if (8 * (r >> 2) + (r & 3) >= lim) sc[r] = -INFINITY;
  }
  float tmax = max3(sc[0], sc[1], sc[2]);
#pragma unroll
  for (int r = 3; r < 15; r += 2) tmax = max3(tmax, sc[r], sc[r + 1]);
  tmax = pair_max(max2(tmax, sc[15]));
  // O and l are rescaled only when some row's max exceeds its reference by
  // more than kLazyLog2 (log2 units): the weights then stay below 2^kLazyLog2
  // and after the first tiles almost every step skips the multiplies. l sums
  // the unrounded weights in fp32, so the LSE is unaffected by the bf16
  // rounding of the weights.
  if (__any(tmax > w.m_run + w.lazy)) {
    const float m_new = fmaxf(w.m_run, tmax);
    const float alpha = exp2_hw((w.m_run - m_new) * a.scale_log2);
    w.l_run *= alpha;
    w.lr_run *= alpha;
#pragma unroll
    for (int db = 0; db < C::dBlocks; ++db) w.acc[db] *= alpha;
    w.m_run = m_new;
  }
  const float mc = w.m_run * a.scale_log2;
#pragma unroll
  for (int r = 0; r < 16; ++r) sc[r] = exp2_hw(fmaf(sc[r], a.scale_log2, -mc));
  float s0 = sc[0] + sc[1], s1 = sc[2] + sc[3];
#pragma unroll
  for (int r = 4; r < 16; r += 4) {
    s0 += sc[r] + sc[r + 1];
    s1 += sc[r + 2] + sc[r + 3];
  }
  w.l_run += s0 + s1;
  bf16x8 pf0, pf1;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    pf0[e] = (__bf16)sc[e];
    pf1[e] = (__bf16)sc[8 + e];
  }
  // O is normalised by the sum of the weights the P V MFMAs actually apply, so
  // the bf16 rounding of a dominant weight cancels in the quotient
  {
    const bf16x2 one2 = {(__bf16)1.f, (__bf16)1.f};
    float r0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pf0, pf0, 0, 1), one2, w.lr_run, false);
    float r1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pf0, pf0, 2, 3), one2, 0.f, false);
    r0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pf0, pf0, 4, 5), one2, r0, false);
    r1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pf0, pf0, 6, 7), one2, r1, false);
    r0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pf1, pf1, 0, 1), one2, r0, false);
    r1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pf1, pf1, 2, 3), one2, r1, false);
    r0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pf1, pf1, 4, 5), one2, r0, false);
    r1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pf1, pf1, 6, 7), one2, r1, false);
    w.lr_run = r0 + r1;
  }
  // O^T += V^T . P^T over the two slices
  bf16x8 vf[C::dBlocks];
  tr_wait<2 * C::dBlocks, C::dBlocks>(v0, vf);
#pragma unroll
  for (int db = 0; db < C::dBlocks; ++db) w.acc[db] = mfma32(vf[db], pf0, w.acc[db]);
  if constexpr (B == 0) {
    // the second half's K operands, in flight during the last MFMAs (tmax
    // depends on this half's S^T MFMAs, which have read the old ones)
    k_issue<C::kSlices, BUF * 2 * C::tileBytes + 32 * C::rowBytes>(w.koff, w.kr, tmax);
    tr_wait<C::kSlices, C::dBlocks>(v1, vf);
  } else {
    tr_wait<0, C::dBlocks>(v1, vf);
  }
#pragma unroll
  for (int db = 0; db < C::dBlocks; ++db) w.acc[db] = mfma32(vf[db], pf1, w.acc[db]);
}

// One 64-key tile (nv valid keys) from LDS buffer BUF; the next tile of the
// piece (ending at t_end) is loaded into the other buffer while the first K
// operands are in flight. Returns the next tile's number of valid keys.
template <int D, int BUF>
__device__ __forceinline__ int tile_step(const AttnArgs& a, Wave<D>& w, const Loop& L, char* smem, int t, int nv,
                                         int t_end) {
  using C = Cfg<D>;
  // half 0's K operands: the tile became visible at the last barrier
  k_issue<C::kSlices, BUF * 2 * C::tileBytes>(w.koff, w.kr, 0.f);
  int n1 = 0;
  if (t + 1 < t_end) {
    int64_t k1;
    tile_of(L.map, t + 1, k1, n1);
    stage_tile<D>(a, k1 * a.ld + L.hoff, n1, smem + (BUF ^ 1) * 2 * C::tileBytes, w.voffk, w.voffv, L.wave);
  }
  half_step<D, BUF, 0>(a, w, L, smem, nv);
  // the last P V MFMAs of half 0 are issued before half 1 waits for its K
  __builtin_amdgcn_sched_barrier(0);
  half_step<D, BUF, 1>(a, w, L, smem, nv);
  __builtin_amdgcn_s_waitcnt(0);  // the next tile's direct loads have landed
  __syncthreads();
  return n1;
}

// Segment arithmetic of the split (shared by the attention and merge kernels).
__device__ __forceinline__ int64_t seg_begin(const AttnSplit& s, int g) { return (int64_t)g * s.units / s.n_seg; }
// segment that holds unit u: the largest g with seg_begin(g) <= u
__device__ __forceinline__ int seg_of(const AttnSplit& s, int64_t u) {
  return (int)(((u + 1) * s.n_seg - 1) / s.units);
}

// One piece: tiles [ta, tb) of work item `item` with a fresh softmax state.
// Whatever the piece completes (all tiles, or all local tiles from tile 0) is
// written to the outputs; the rest goes to partial slot `slot`.
template <int D>
__device__ __forceinline__ void run_piece(const AttnArgs& a, Wave<D>& w, Loop& L, char* smem, int q_tiles, int item,
                                          int ta, int tb, int slot, int ql) {
  using C = Cfg<D>;
  const int head = item / q_tiles;
  const int qtile = item - head * q_tiles;
  L.hoff = head * D;
  const int qloc = L.wave * kBqWave + ql;
  const int qrow = qtile * kBq + qloc;
  // ---- Q^T operand, resident for the piece -----------------------------------
  {
    const uint16_t* qp = a.q + (int64_t)qrow * a.ld + L.hoff + 8 * L.hh;
#pragma unroll
    for (int kk = 0; kk < C::kSlices; ++kk) w.qf[kk] = qrow < a.n_q ? *(const bf16x8*)(qp + 16 * kk) : bf16x8{};
  }
#pragma unroll
  for (int i = 0; i < C::dBlocks; ++i) w.acc[i] = f32x16{};
  w.m_run = -INFINITY;
  w.l_run = 0.f;
  w.lr_run = 0.f;

  int nv;  // valid keys of the tile in the current buffer
  {
    int64_t k0;
    tile_of(L.map, ta, k0, nv);
    stage_tile<D>(a, k0 * a.ld + L.hoff, nv, smem, w.voffk, w.voffv, L.wave);
  }
  __builtin_amdgcn_s_waitcnt(0);  // this wave's direct loads have landed
  __syncthreads();

  const int Lt = L.n_tiles_local;
  for (int t = ta; t < tb; t += 2) {
    // local set complete after tile Lt - 1 (a piece that started at tile 0 owns it)
    if (L.dual && t == Lt && t > ta)
      write_state<D>(a, w, L, qloc, qrow, head, a.out_local, a.lse_local, ta == 0 ? -1 : slot, 1);
    nv = tile_step<D, 0>(a, w, L, smem, t, nv, tb);
    if (t + 1 < tb) {
      if (L.dual && t + 1 == Lt)
        write_state<D>(a, w, L, qloc, qrow, head, a.out_local, a.lse_local, ta == 0 ? -1 : slot, 1);
      nv = tile_step<D, 1>(a, w, L, smem, t + 1, nv, tb);
    }
  }
  const bool whole = ta == 0 && tb == L.n_tiles;
  write_state<D>(a, w, L, qloc, qrow, head, a.out, a.lse, whole ? -1 : slot, 0);
  // a piece ending inside (or at the end of) the local set also holds its
  // local contribution
  if (L.dual && tb <= Lt)
    write_state<D>(a, w, L, qloc, qrow, head, a.out_local, a.lse_local, (ta == 0 && tb == Lt) ? -1 : slot, 1);
}

template <int D>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2))) void attn_chunk_kernel(AttnArgs a,
                                                                                                  int q_tiles) {
  using C = Cfg<D>;
  __shared__ __attribute__((aligned(1024))) char smem[2 * 2 * C::tileBytes];  // [buf][K|V]

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  Loop L;
  L.wave = tid >> 6;
  L.hh = lane >> 5;  // lane half
  const int ql = lane & 31;  // this lane's query within the wave

  // ---- tile enumeration (the same for every work item) --------------------------
  const int nt0 = (int)((a.r.end[0] - a.r.begin[0] + kBk - 1) / kBk);
  const int nt1 = a.r.n_total > 1 ? (int)((a.r.end[1] - a.r.begin[1] + kBk - 1) / kBk) : 0;
  const int nt2 = a.r.n_total > 2 ? (int)((a.r.end[2] - a.r.begin[2] + kBk - 1) / kBk) : 0;
  L.map.b0 = a.r.begin[0];
  L.map.e0 = a.r.end[0];
  L.map.b1 = a.r.n_total > 1 ? a.r.begin[1] : 0;
  L.map.e1 = a.r.n_total > 1 ? a.r.end[1] : 0;
  L.map.b2 = a.r.n_total > 2 ? a.r.begin[2] : 0;
  L.map.e2 = a.r.n_total > 2 ? a.r.end[2] : 0;
  L.map.tb1 = a.r.n_total > 1 ? nt0 : INT_MAX;
  L.map.tb2 = a.r.n_total > 2 ? nt0 + nt1 : INT_MAX;
  L.n_tiles = nt0 + nt1 + nt2;
  L.n_tiles_local = a.r.n_local == 1 ? nt0 : nt0 + nt1;
  L.dual = a.out_local != nullptr;
  const int T = L.n_tiles;
  if (T <= 0) return;  // (an empty key set is handled on the host)

  // ---- XCD-aware mapping of workgroups to work items or segments ------------------
  // The 8 XCDs take workgroups round-robin; consecutive logical indices (the
  // tiles of one head) stay on one XCD and share its L2.
  const int n_work = q_tiles * a.n_heads;
  const int n_log = a.split.n_seg > 0 ? a.split.n_seg : n_work;
  const int per_xcd = (int)(gridDim.x / kXcds);
  const int bid = blockIdx.x;
  const int g = (bid % kXcds) * per_xcd + bid / kXcds;
  if (g >= n_log) return;  // padding blocks (uniform exit, before any barrier)
  int64_t u0, u1;
  if (a.split.n_seg > 0) {
    u0 = seg_begin(a.split, g);
    u1 = seg_begin(a.split, g + 1);
  } else {
    u0 = (int64_t)g * T;
    u1 = u0 + T;
  }

  Wave<D> w;
  // ---- per-lane constants ---------------------------------------------------------
  // Direct load q of this thread covers 16-byte slot (q * kWaves + wave) * 64 + lane
  // of a tile: row = slot / chunksPerRow, stored chunk = slot % chunksPerRow,
  // which holds logical chunk (stored ^ swizzle(row)) of that key row.
  {
    const int slot = L.wave * 64 + lane;
    const int row = slot / C::chunksPerRow;
    const int stored = slot % C::chunksPerRow;
    w.voffk = (int)((row * a.ld + (stored ^ swz_k<D>(row)) * 8) * 2);
    w.voffv = (int)((row * a.ld + (stored ^ swz_v<D>(row)) * 8) * 2);
  }
  {
    const uint32_t lds0 = lds_addr(smem);
#pragma unroll
    for (int kk = 0; kk < C::kSlices; ++kk) w.koff[kk] = lds0 + chunk_off<D>(ql, 2 * kk + L.hh, swz_k<D>(ql));
    const int gq = lane >> 4, sl = lane & 15;
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
      for (int db = 0; db < C::dBlocks; ++db) {
        const int row = 8 * h2 + 4 * (gq >> 1) + (sl >> 2);
        const int chunk = 4 * db + 2 * (gq & 1) + ((sl & 3) >> 1);
        w.vaddr[h2][db] = lds0 + chunk_off<D>(row, chunk, swz_v<D>(row)) + ((sl & 1) << 3);
      }
  }
  w.lazy = kLazyLog2 / a.scale_log2;

  // ---- the pieces of this workgroup's unit range, last one first -------------------
  // The last piece starts at tile 0 of its item and the first one ends at the
  // item's last tile, so with this order every segment of a head visits the
  // same tile offset at the same time (from the start, then from the end of
  // the item): the workgroups of one head keep sharing K/V through L2.
  const int i_first = (int)(u0 / T), i_last = (int)((u1 - 1) / T);
  for (int item = i_last; item >= i_first; --item) {
    const int64_t ibase = (int64_t)item * T;
    const int ta = (int)((u0 > ibase ? u0 : ibase) - ibase);
    const int tb = (int)((u1 < ibase + T ? u1 : ibase + T) - ibase);
    run_piece<D>(a, w, L, smem, q_tiles, item, ta, tb,
                 a.split.n_seg > 0 ? g * a.split.max_pieces + (item - i_first) : -1, ql);
  }
}

// Eq. 11-12 over the pieces of each split work item: for every query row,
// LSE = m + ln sum_p e^(LSE_p - m) and O = sum_p e^(LSE_p - LSE) O_p, for the
// full result (all pieces) and the local result (pieces that start in the local
// set). Items or sets covered by one piece were written by that piece.
// floor(n / d) for 0 <= n < 2^53 and 0 < d in fp64: n and d are exact, and a
// quotient q that is not an integer lies at least 1/d from one, farther than
// the rounding of the division (at most q 2^-53 < 1/d) can move it, so the
// floor is exact.
__device__ __forceinline__ int64_t floor_div_exact(int64_t n, int64_t d) {
  return (int64_t)__builtin_floor((double)n / (double)d);
}

template <int D>
__global__ __launch_bounds__(256) void attn_merge_split_kernel(AttnArgs a, int q_tiles, int n_tiles,
                                                               int n_tiles_local) {
  constexpr int kVec = D / 4;            // float4 per row
  constexpr int kRows = 256 / kVec;      // rows per block
  constexpr int kBatch = 4;              // pieces whose loads are in flight together
  const AttnSplit& s = a.split;
  const int item = blockIdx.x;
  const int r = threadIdx.x / kVec, c = threadIdx.x % kVec;
  const int qloc = blockIdx.y * kRows + r;
  const int head = item / q_tiles;
  const int qrow = (item - head * q_tiles) * kBq + qloc;
  if (qrow >= a.n_q) return;
  // segments g_lo .. g_hi hold the pieces of this item: the same arithmetic as
  // seg_of / seg_begin, exact in fp64 since units x segments < 2^52 (checked
  // on the host)
  const int64_t i0 = (int64_t)item * n_tiles;
  const int g_lo = (int)floor_div_exact((i0 + 1) * s.n_seg - 1, s.units);
#pragma unroll
  for (int which = 0; which < 2; ++which) {
    if (which == 1 && a.out_local == nullptr) break;
    const int64_t u_last = i0 + (which == 0 ? n_tiles : n_tiles_local) - 1;
    const int g_hi = (int)floor_div_exact((u_last + 1) * s.n_seg - 1, s.units);
    if (g_hi == g_lo) continue;
    // Eq. 11-12 over the pieces, kBatch at a time with a running maximum
    float m = -INFINITY, sum = 0.f;
    f32x4 o = {0.f, 0.f, 0.f, 0.f};
    for (int g0 = g_lo; g0 <= g_hi; g0 += kBatch) {
      float l[kBatch];
      f32x4 v[kBatch];
#pragma unroll
      for (int j = 0; j < kBatch; ++j) {
        const int gg = g0 + j;
        l[j] = -INFINITY;
        v[j] = f32x4{0.f, 0.f, 0.f, 0.f};
        if (gg <= g_hi) {
          const int64_t first = floor_div_exact(floor_div_exact((int64_t)gg * s.units, s.n_seg), n_tiles);
          const int slot = gg * s.max_pieces + (item - (int)first);
          const int64_t base = ((int64_t)slot * 2 + which) * kBq + qloc;
          l[j] = s.part_lse[base];
          v[j] = *(const f32x4*)(s.part_o + base * D + 4 * c);
        }
      }
      float mm = m;
#pragma unroll
      for (int j = 0; j < kBatch; ++j) mm = fmaxf(mm, l[j]);
      const float sc = m == -INFINITY ? 0.f : expf(m - mm);
      sum *= sc;
      o *= sc;
#pragma unroll
      for (int j = 0; j < kBatch; ++j) {
        const float e = l[j] == -INFINITY ? 0.f : expf(l[j] - mm);
        sum += e;
        o += e * v[j];
      }
      m = mm;
    }
    const float inv = 1.f / sum;
    float* out = which == 0 ? a.out : a.out_local;
    float* lse = which == 0 ? a.lse : a.lse_local;
    *(f32x4*)(out + (int64_t)qrow * a.ld + (int64_t)head * D + 4 * c) = o * inv;
    if (lse != nullptr && c == 0) lse[(int64_t)head * a.n_q + qrow] = m + logf(sum);
  }
}

// Attention over an empty key set: O = 0, LSE = -inf (the convention that
// makes Eq. 11-12 return the other branch unchanged).
__global__ void attn_empty_kernel(float* out, float* lse, int64_t n_out, int64_t n_lse) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_out; i += (int64_t)gridDim.x * blockDim.x) {
    out[i] = 0.f;
    if (lse != nullptr && i < n_lse) lse[i] = -INFINITY;
  }
}

// Eq. 11-12 for two results over disjoint key sets, evaluated as
// m + ln(e^(a - m) + e^(b - m)); both empty gives O = 0, LSE = -inf.
__global__ void attn_merge2_kernel(const float* o_a, const float* lse_a, const float* o_b, const float* lse_b,
                                   int64_t n_q, int64_t n_heads, int head_dim, float* out, float* lse) {
  const int64_t hidden = n_heads * head_dim;
  const int64_t n4 = n_q * hidden / 4;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t e = 4 * i;
    const int64_t row = e / hidden;
    const int64_t h = (e - row * hidden) / head_dim;
    const float la = lse_a[h * n_q + row], lb = lse_b[h * n_q + row];
    const float m = fmaxf(la, lb);
    f32x4 o = {0.f, 0.f, 0.f, 0.f};
    float l = -INFINITY;
    if (m != -INFINITY) {
      const float ea = expf(la - m), eb = expf(lb - m);
      l = m + logf(ea + eb);
      const float wa = expf(la - l), wb = expf(lb - l);
      const f32x4 va = *(const f32x4*)(o_a + e), vb = *(const f32x4*)(o_b + e);
      o = wa * va + wb * vb;
    }
    *(f32x4*)(out + e) = o;
    if (lse != nullptr && e % head_dim == 0) lse[h * n_q + row] = l;
  }
}

}  // namespace

int attn_tiles(const AttnRanges& r, int* n_tiles_local) {
  int nt[3] = {0, 0, 0};
  for (int i = 0; i < r.n_total; ++i) nt[i] = (int)((r.end[i] - r.begin[i] + kBk - 1) / kBk);
  if (n_tiles_local) *n_tiles_local = r.n_local == 1 ? nt[0] : nt[0] + nt[1];
  return nt[0] + nt[1] + nt[2];
}

int attn_cu_count() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  static int cache[64];
  if (dev >= 0 && dev < 64 && cache[dev] > 0) return cache[dev];
  int n = 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  if (dev >= 0 && dev < 64) cache[dev] = n;
  return n;
}

size_t attn_plan_split(const AttnArgs& a, int head_dim, int segments, AttnSplit* s) {
  s->units = 0;
  s->n_seg = 0;
  s->max_pieces = 0;
  s->part_o = nullptr;
  s->part_lse = nullptr;
  s->ctr = nullptr;
  s->lse_offset = s->ctr_offset = 0;
  const int T = attn_tiles(a.r, nullptr);
  const int64_t n_work = (int64_t)((a.n_q + kBq - 1) / kBq) * a.n_heads;
  if (segments < 0 || T <= 0) return 0;
  const int64_t U = n_work * T;
  int64_t G;
  if (segments > 0) {
    G = segments;
  } else {
    // whole work items per workgroup leave a fraction of the last round of
    // workgroups idle; split only when that fraction is large and the launch
    // is long enough to repay the partial results' traffic and the merge.
    // The chip runs these launches at its power limit, where idle compute
    // units let the busy ones clock higher: 228 items on 256 CUs (89% full)
    // take as long whole as split, with 40% fewer HBM bytes; at 82% and
    // below the split is faster (ISPA_ATTN_SPLIT_FILL overrides the percent)
    const int n_cu = attn_cu_count();
    if (n_cu <= 0 || T < kSplitMinTiles) return 0;
    const int64_t rounds = (n_work + n_cu - 1) / n_cu;
    const char* fill_env = getenv("ISPA_ATTN_SPLIT_FILL");
    const int fill_pct = fill_env != nullptr ? atoi(fill_env) : kSplitFillPct;
    if (n_work * 100 >= rounds * n_cu * fill_pct) return 0;
    G = n_cu;
    if (U / G < 16) G = U / 16;
    if (G < 2) return 0;
  }
  if (G > U) G = U;
  if (G > (1 << 20)) G = 1 << 20;
  // the merge kernel's segment arithmetic is exact in fp64 below 2^52
  while (G > 1 && (double)U * (double)G >= 4503599627370496.0) G /= 2;
  const int64_t seg_max = (U + G - 1) / G;
  s->units = U;
  s->n_seg = (int32_t)G;
  s->max_pieces = (int32_t)((seg_max + T - 1) / T + 1);
  const size_t slots = (size_t)G * s->max_pieces * 2 * kBq;
  s->lse_offset = (slots * head_dim * 4 + 255) / 256 * 256;
  s->ctr_offset = (s->lse_offset + slots * 4 + 255) / 256 * 256;
  return s->ctr_offset + (size_t)n_work * 2 * 4 * sizeof(uint32_t);
}

hipError_t launch_attn_chunk(const AttnArgs& a, int head_dim, hipStream_t stream) {
  const int q_tiles = (a.n_q + kBq - 1) / kBq;
  const int n_work = q_tiles * a.n_heads;
  const int n_log = a.split.n_seg > 0 ? a.split.n_seg : n_work;
  const int per_xcd = (n_log + kXcds - 1) / kXcds;
  const int grid = per_xcd * kXcds;
  hipError_t e;
  if (attn_fast_eligible(a, head_dim)) {
    // split: the pieces complete their work items (counters cleared first);
    // no merge kernel (ISPA_ATTN_MERGE_KERNEL=1: the merge kernel instead)
    const char* env = getenv("ISPA_ATTN_MERGE_KERNEL");
    if (a.split.n_seg > 0 && a.split.ctr != nullptr && !(env != nullptr && env[0] == '1')) {
      e = launch_zero(a.split.ctr, (size_t)n_work * 2 * 4 * sizeof(uint32_t), stream);
      if (e != hipSuccess) return e;
      return launch_attn_fast(a, stream);
    }
    e = launch_attn_fast(a, stream);
  } else {
    if (head_dim == 128) {
      hipLaunchKernelGGL(attn_chunk_kernel<128>, dim3(grid), dim3(kThreads), 0, stream, a, q_tiles);
    } else {
      hipLaunchKernelGGL(attn_chunk_kernel<64>, dim3(grid), dim3(kThreads), 0, stream, a, q_tiles);
    }
    e = hipGetLastError();
  }
  if (e != hipSuccess || a.split.n_seg == 0) return e;
  int n_local = 0;
  const int T = attn_tiles(a.r, &n_local);
  const dim3 mgrid(n_work, head_dim == 128 ? kBq / 8 : kBq / 16);
  if (head_dim == 128) {
    hipLaunchKernelGGL(attn_merge_split_kernel<128>, mgrid, dim3(256), 0, stream, a, q_tiles, T, n_local);
  } else {
    hipLaunchKernelGGL(attn_merge_split_kernel<64>, mgrid, dim3(256), 0, stream, a, q_tiles, T, n_local);
  }
  return hipGetLastError();
}

hipError_t launch_attn_empty(float* out, float* lse, int64_t n_q, int64_t n_heads, int head_dim,
                             hipStream_t stream) {
  const int64_t n_out = n_q * n_heads * head_dim;
  const int blocks = (int)((n_out + 255) / 256 < 4096 ? (n_out + 255) / 256 : 4096);
  hipLaunchKernelGGL(attn_empty_kernel, dim3(blocks), dim3(256), 0, stream, out, lse, n_out, n_q * n_heads);
  return hipGetLastError();
}

hipError_t launch_attn_merge2(const float* o_a, const float* lse_a, const float* o_b, const float* lse_b,
                              int64_t n_q, int64_t n_heads, int head_dim, float* out, float* lse,
                              hipStream_t stream) {
  const int64_t n4 = n_q * n_heads * head_dim / 4;
  const int blocks = (int)((n4 + 255) / 256 < 8192 ? (n4 + 255) / 256 : 8192);
  hipLaunchKernelGGL(attn_merge2_kernel, dim3(blocks), dim3(256), 0, stream, o_a, lse_a, o_b, lse_b, n_q, n_heads,
                     head_dim, out, lse);
  return hipGetLastError();
}

}  // namespace ispa
