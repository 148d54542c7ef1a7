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
//   workgroup = 4 waves = 128 queries of one head; each wave owns 32 queries.
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
//   p = 2^(s * c - m * c), c = scale * log2(e); LSE = m * scale + ln(l).
//
// Workgroups are remapped so that the 8 XCDs (dispatched round-robin) each own
// a contiguous run of (head, query tile) work items: tiles of one head share
// the K/V stream through one XCD's L2.
#include "ispa_internal.h"

#include <math.h>

namespace ispa {
namespace {

constexpr int kWaves = 4;
constexpr int kThreads = kWaves * 64;
constexpr int kBqWave = 32;
constexpr int kBq = kWaves * kBqWave;  // queries per workgroup
constexpr int kBk = 64;                // keys per tile
constexpr int kXcds = 8;

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

// LDS transpose reads of one 16-key slice for all dBlocks column blocks (two
// reads per block), issued as inline asm and completed by an explicit wait that
// is tied to their results. Through the builtin the compiler cannot tell these
// reads from reads of the buffer the direct loads are filling, and would wait
// for those loads (vmcnt 0) before every slice. LDS operations complete in
// order, so the compiler's own lgkmcnt waits stay correct around these.
__device__ __forceinline__ uint32_t lds_addr(const char* p) {
  return (uint32_t)(uintptr_t)(ISPA_LDS const char*)p;
}
template <int NB>
__device__ __forceinline__ void lds_read_tr_slice(const char* base, const int (*off)[NB], bf16x8* out) {
  u32x2 r0[NB], r1[NB];
#pragma unroll
  for (int db = 0; db < NB; ++db) {
    asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(r0[db]) : "v"(lds_addr(base + off[0][db])));
    asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(r1[db]) : "v"(lds_addr(base + off[1][db])));
  }
#pragma unroll
  for (int db = 0; db < NB; ++db) asm volatile("" : "+v"(r0[db]), "+v"(r1[db]));
  if constexpr (NB == 4) {
    asm volatile("s_waitcnt lgkmcnt(0)"
                 : "+v"(r0[0]), "+v"(r1[0]), "+v"(r0[1]), "+v"(r1[1]), "+v"(r0[2]), "+v"(r1[2]), "+v"(r0[3]),
                   "+v"(r1[3]));
  } else {
    asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(r0[0]), "+v"(r1[0]), "+v"(r0[1]), "+v"(r1[1]));
  }
#pragma unroll
  for (int db = 0; db < NB; ++db) {
    const u32x4 w{r0[db][0], r0[db][1], r1[db][0], r1[db][1]};
    out[db] = __builtin_bit_cast(bf16x8, w);
  }
}

// Tile t of the flattened range list: first key and number of valid keys.
// tb1/tb2 are the tile indices where ranges 1 and 2 start.
__device__ __forceinline__ void tile_of(const AttnRanges& r, int tb1, int tb2, int t,
                                        int64_t& key0, int& nvalid) {
  const bool in2 = r.n_total > 2 && t >= tb2;
  const bool in1 = !in2 && r.n_total > 1 && t >= tb1;
  const int64_t begin = in2 ? r.begin[2] : (in1 ? r.begin[1] : r.begin[0]);
  const int64_t end = in2 ? r.end[2] : (in1 ? r.end[1] : r.end[0]);
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
                                           const int* voffk, const int* voffv, int wave) {
  using C = Cfg<D>;
  const int nbytes = (int)(((int64_t)(nv - 1) * a.ld + D) * 2);
  const __amdgpu_buffer_rsrc_t rk = make_rsrc(a.k + base, nbytes);
  const __amdgpu_buffer_rsrc_t rv = make_rsrc(a.v + base, nbytes);
#pragma unroll
  for (int q = 0; q < C::loadsPerThread; ++q) {
    const int wslot = (q * kWaves + wave) * 64 * 16;  // wave-uniform LDS destination
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, (ISPA_LDS void*)(dst + wslot), 16, voffk[q], 0, 0, 0);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, (ISPA_LDS void*)(dst + C::tileBytes + wslot), 16, voffv[q], 0,
                                             0, 0);
  }
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
  const int wave = tid >> 6;
  const int ql = lane & 31;  // this lane's query within the wave
  const int hh = lane >> 5;  // lane half
  const int64_t ld = a.ld;
  const int hoff = head * D;
  const int qrow = qtile * kBq + wave * kBqWave + ql;
  const bool q_ok = qrow < a.n_q;

  // ---- Q^T operand, resident for the whole key loop ------------------------
  bf16x8 qf[C::kSlices];
  {
    const uint16_t* qp = a.q + (int64_t)qrow * ld + hoff + 8 * hh;
#pragma unroll
    for (int kk = 0; kk < C::kSlices; ++kk) {
      if (q_ok) {
        qf[kk] = *(const bf16x8*)(qp + 16 * kk);
      } else {
        qf[kk] = bf16x8{};
      }
    }
  }

  // ---- tile enumeration -------------------------------------------------------
  const int nt0 = (int)((a.r.end[0] - a.r.begin[0] + kBk - 1) / kBk);
  const int nt1 = a.r.n_total > 1 ? (int)((a.r.end[1] - a.r.begin[1] + kBk - 1) / kBk) : 0;
  const int nt2 = a.r.n_total > 2 ? (int)((a.r.end[2] - a.r.begin[2] + kBk - 1) / kBk) : 0;
  const int tb1 = nt0, tb2 = nt0 + nt1;
  const int n_tiles = nt0 + nt1 + nt2;
  const int n_tiles_local = a.r.n_local == 1 ? nt0 : nt0 + nt1;
  const bool dual = a.out_local != nullptr;

  // ---- online softmax state ------------------------------------------------------
  f32x16 acc[C::dBlocks];
#pragma unroll
  for (int i = 0; i < C::dBlocks; ++i) acc[i] = f32x16{};
  float m_run = -INFINITY;
  float l_run = 0.f;

  // ---- HBM -> LDS staging ------------------------------------------------
  // Load q of this thread covers 16-byte slot (q * kWaves + wave) * 64 + lane of
  // the tile: row = slot / chunksPerRow, stored chunk = slot % chunksPerRow,
  // which holds logical chunk (stored ^ (row & swz)) of that key row.
  int voffk[C::loadsPerThread], voffv[C::loadsPerThread];
#pragma unroll
  for (int q = 0; q < C::loadsPerThread; ++q) {
    const int slot = (q * kWaves + wave) * 64 + lane;
    const int row = slot / C::chunksPerRow;
    const int stored = slot % C::chunksPerRow;
    voffk[q] = (int)((row * ld + (stored ^ swz_k<D>(row)) * 8) * 2);
    voffv[q] = (int)((row * ld + (stored ^ swz_v<D>(row)) * 8) * 2);
  }
  auto gload = [&](int t, int buf) {
    int64_t key0;
    int nv;
    tile_of(a.r, tb1, tb2, t, key0, nv);
    stage_tile<D>(a, key0 * ld + hoff, nv, smem + buf * 2 * C::tileBytes, voffk, voffv, wave);
  };

  // per-lane LDS byte offsets of the MFMA operands (tile-relative)
  int koff[C::kSlices];
#pragma unroll
  for (int kk = 0; kk < C::kSlices; ++kk) koff[kk] = chunk_off<D>(ql, 2 * kk + hh, swz_k<D>(ql));
  const int g = lane >> 4;
  const int sl = lane & 15;
  int voffr[2][C::dBlocks];
#pragma unroll
  for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
    for (int db = 0; db < C::dBlocks; ++db) {
      const int row = 8 * h2 + 4 * (g >> 1) + (sl >> 2);
      const int chunk = 4 * db + 2 * (g & 1) + ((sl & 3) >> 1);
      voffr[h2][db] = chunk_off<D>(row, chunk, swz_v<D>(row)) + ((sl & 1) << 3);
    }

  auto finish = [&](float* out, float* lse) {
    const float l_tot = l_run + __shfl_xor(l_run, 32);
    const float inv = 1.0f / l_tot;
    if (q_ok) {
      float* op = out + (int64_t)qrow * ld + hoff + 4 * hh;
#pragma unroll
      for (int db = 0; db < C::dBlocks; ++db) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          f32x4 o;
          o[0] = acc[db][4 * i + 0] * inv;
          o[1] = acc[db][4 * i + 1] * inv;
          o[2] = acc[db][4 * i + 2] * inv;
          o[3] = acc[db][4 * i + 3] * inv;
          *(f32x4*)(op + 32 * db + 8 * i) = o;
        }
      }
      if (lse != nullptr && hh == 0) lse[(int64_t)head * a.n_q + qrow] = m_run * a.scale + logf(l_tot);
    }
  };

  if (n_tiles > 0) gload(0, 0);
  __builtin_amdgcn_s_waitcnt(0);  // this wave's direct loads have landed
  __syncthreads();

  for (int t = 0; t < n_tiles; ++t) {
    const int buf = t & 1;
    if (dual && t == n_tiles_local) finish(a.out_local, a.lse_local);
    int64_t key0;
    int nv;
    tile_of(a.r, tb1, tb2, t, key0, nv);
    if (t + 1 < n_tiles) gload(t + 1, buf ^ 1);

    const char* ks = smem + buf * 2 * C::tileBytes;
    const char* vs = ks + C::tileBytes;

    // The tile is processed as two halves of 32 keys; each half is a complete
    // online-softmax step (scores, max, lazy rescale, exp, P.V), which keeps
    // only 16 score registers live.
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      // S^T = K . Q^T for keys 32b .. 32b+31 (rows 32b + ql share the swizzle of row ql)
      f32x16 sc = f32x16{};
      const char* kp = ks + 32 * b * C::rowBytes;
#pragma unroll
      for (int kk = 0; kk < C::kSlices; ++kk) {
        const bf16x8 kf = *(const bf16x8*)(kp + koff[kk]);
        sc = mfma32(kf, qf[kk], sc);
      }
      // mask keys beyond the end of a range (only the last tile of each range)
      if (nv < 32 * (b + 1)) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = 32 * b + 8 * (r >> 2) + 4 * hh + (r & 3);
          if (key >= nv) sc[r] = -INFINITY;
        }
      }
      float tmax = fmaxf(sc[0], sc[1]);
#pragma unroll
      for (int r = 2; r < 16; ++r) tmax = fmaxf(tmax, sc[r]);
      tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
      // O and l are rescaled only when some row's running max grew: after the
      // first few tiles most halves skip the 64 multiplies. The reference stays
      // the exact running max, so the largest weight of a row is exactly 1 and
      // carries no bf16 rounding error (a stale reference would put rounding
      // error on the dominant terms).
      if (__any(tmax > m_run)) {
        const float m_new = fmaxf(m_run, tmax);
        const float alpha = exp2_hw((m_run - m_new) * a.scale_log2);
        l_run *= alpha;
#pragma unroll
        for (int db = 0; db < C::dBlocks; ++db) acc[db] *= alpha;
        m_run = m_new;
      }
      const float mc = m_run * a.scale_log2;
      float psum = 0.f;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = exp2_hw(fmaf(sc[r], a.scale_log2, -mc));
        sc[r] = p;
        psum += p;
      }
      l_run += psum;
      // O^T += V^T . P^T over the two 16-key slices of this half
#pragma unroll
      for (int t2 = 0; t2 < 2; ++t2) {
        bf16x8 pf;
#pragma unroll
        for (int e = 0; e < 8; ++e) pf[e] = (__bf16)sc[8 * t2 + e];
        // rows 16 * slice + ...: both swizzles repeat every 16 rows
        const char* vp = vs + 16 * (2 * b + t2) * C::rowBytes;
        bf16x8 vf[C::dBlocks];
        lds_read_tr_slice<C::dBlocks>(vp, voffr, vf);
#pragma unroll
        for (int db = 0; db < C::dBlocks; ++db) acc[db] = mfma32(vf[db], pf, acc[db]);
      }
    }

    __builtin_amdgcn_s_waitcnt(0);  // the next tile's direct loads have landed
    __syncthreads();
  }

  if (dual && n_tiles_local == n_tiles) finish(a.out_local, a.lse_local);
  finish(a.out, a.lse);
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
