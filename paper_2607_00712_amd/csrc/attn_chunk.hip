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
#include "ispa_internal.h"

#include <limits.h>
#include <math.h>

namespace ispa {
namespace {

constexpr int kWaves = 8;
constexpr int kThreads = kWaves * 64;
constexpr int kBqWave = 32;
constexpr int kBq = kWaves * kBqWave;  // queries per workgroup
constexpr int kBk = 64;                // keys per tile
constexpr int kXcds = 8;
constexpr float kLazyLog2 = 8.f;       // rescale threshold of the softmax reference

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
  float l_run;                 // running sum of p (this lane's half of the keys)
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

template <int D>
__device__ __forceinline__ void finish(const AttnArgs& a, Wave<D>& w, const Loop& L, int qrow, int head,
                                       float* out, float* lse) {
  using C = Cfg<D>;
  const float l_tot = l_run_total(w.l_run);
  const float inv = 1.0f / l_tot;
  if (qrow < a.n_q) {
    float* op = out + (int64_t)qrow * a.ld + L.hoff + 4 * L.hh;
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
    if (lse != nullptr && L.hh == 0) lse[(int64_t)head * a.n_q + qrow] = w.m_run * a.scale + logf(l_tot);
  }
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
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int key = 32 * B + 8 * (r >> 2) + 4 * L.hh + (r & 3);
      if (key >= nv) sc[r] = -INFINITY;
    }
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

// One 64-key tile (nv valid keys) from LDS buffer BUF; the next tile's direct
// loads into the other buffer are issued while the first K operands are in
// flight. Returns the next tile's number of valid keys.
template <int D, int BUF>
__device__ __forceinline__ int tile_step(const AttnArgs& a, Wave<D>& w, const Loop& L, char* smem, int t, int nv) {
  using C = Cfg<D>;
  // half 0's K operands: the tile became visible at the last barrier
  k_issue<C::kSlices, BUF * 2 * C::tileBytes>(w.koff, w.kr, 0.f);
  int n1 = 0;
  if (t + 1 < L.n_tiles) {
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

template <int D>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2))) void attn_chunk_kernel(AttnArgs a,
                                                                                                  int q_tiles) {
  using C = Cfg<D>;
  __shared__ __attribute__((aligned(1024))) char smem[2 * 2 * C::tileBytes];  // [buf][K|V]

  // ---- XCD-aware work mapping ------------------------------------------
  const int n_work = q_tiles * a.n_heads;
  const int per_xcd = (n_work + kXcds - 1) / kXcds;
  const int bid = blockIdx.x;
  const int work = (bid % kXcds) * per_xcd + bid / kXcds;
  if (work >= n_work) return;  // padding blocks (uniform exit, before any barrier)
  const int head = work / q_tiles;
  const int qtile = work % q_tiles;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  Loop L;
  L.wave = tid >> 6;
  L.hh = lane >> 5;  // lane half
  L.hoff = head * D;
  const int ql = lane & 31;  // this lane's query within the wave
  const int qrow = qtile * kBq + L.wave * kBqWave + ql;

  Wave<D> w;
  // ---- Q^T operand, resident for the whole key loop ------------------------
  {
    const uint16_t* qp = a.q + (int64_t)qrow * a.ld + L.hoff + 8 * L.hh;
#pragma unroll
    for (int kk = 0; kk < C::kSlices; ++kk) w.qf[kk] = qrow < a.n_q ? *(const bf16x8*)(qp + 16 * kk) : bf16x8{};
  }

  // ---- tile enumeration -------------------------------------------------------
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
    const int g = lane >> 4, sl = lane & 15;
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
      for (int db = 0; db < C::dBlocks; ++db) {
        const int row = 8 * h2 + 4 * (g >> 1) + (sl >> 2);
        const int chunk = 4 * db + 2 * (g & 1) + ((sl & 3) >> 1);
        w.vaddr[h2][db] = lds0 + chunk_off<D>(row, chunk, swz_v<D>(row)) + ((sl & 1) << 3);
      }
  }

  // ---- online softmax state ------------------------------------------------------
#pragma unroll
  for (int i = 0; i < C::dBlocks; ++i) w.acc[i] = f32x16{};
  w.m_run = -INFINITY;
  w.l_run = 0.f;
  w.lazy = kLazyLog2 / a.scale_log2;

  int nv = 0;  // valid keys of the tile in the current buffer
  if (L.n_tiles > 0) {
    int64_t k0;
    tile_of(L.map, 0, k0, nv);
    stage_tile<D>(a, k0 * a.ld + L.hoff, nv, smem, w.voffk, w.voffv, L.wave);
  }
  __builtin_amdgcn_s_waitcnt(0);  // this wave's direct loads have landed
  __syncthreads();

  for (int t = 0; t < L.n_tiles; t += 2) {
    if (L.dual && t == L.n_tiles_local) finish<D>(a, w, L, qrow, head, a.out_local, a.lse_local);
    nv = tile_step<D, 0>(a, w, L, smem, t, nv);
    if (t + 1 < L.n_tiles) {
      if (L.dual && t + 1 == L.n_tiles_local) finish<D>(a, w, L, qrow, head, a.out_local, a.lse_local);
      nv = tile_step<D, 1>(a, w, L, smem, t + 1, nv);
    }
  }
  if (L.dual && L.n_tiles_local == L.n_tiles) finish<D>(a, w, L, qrow, head, a.out_local, a.lse_local);
  finish<D>(a, w, L, qrow, head, a.out, a.lse);
}

}  // namespace

hipError_t launch_attn_chunk(const AttnArgs& a, int head_dim, hipStream_t stream) {
  const int q_tiles = (a.n_q + kBq - 1) / kBq;
  const int n_work = q_tiles * a.n_heads;
  const int per_xcd = (n_work + kXcds - 1) / kXcds;
  const int grid = per_xcd * kXcds;
  if (head_dim == 128) {
    hipLaunchKernelGGL(attn_chunk_kernel<128>, dim3(grid), dim3(kThreads), 0, stream, a, q_tiles);
  } else {
    hipLaunchKernelGGL(attn_chunk_kernel<64>, dim3(grid), dim3(kThreads), 0, stream, a, q_tiles);
  }
  return hipGetLastError();
}

}  // namespace ispa
