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
//   Keys are visited in tiles of 64 rows, staged in LDS (double buffered, one
//   barrier per tile). Only tiles that intersect the key set are visited; the
//   tile at the end of each contiguous range is masked element-wise.
//
// Per tile and wave (bf16 MFMA 32x32x16, fp32 accumulation):
//   S^T[64 keys x 32 q] = K_tile . Q^T   -- A = K rows from LDS, B = Q^T in VGPRs.
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
  static constexpr int kStride = D + 8;    // K row stride in LDS (elements)
  static constexpr int vStride = D + 16;   // V row stride in LDS (elements)
  static constexpr int kTile = kBk * kStride;
  static constexpr int vTile = kBk * vStride;
  static constexpr int chunksPerRow = D / 8;                 // 16-byte chunks
  static constexpr int chunksPerThread = kBk * chunksPerRow / kThreads;
  static constexpr int kSlices = D / 16;                     // QK^T k-steps
  static constexpr int dBlocks = D / 32;                     // O^T row blocks
  static_assert(kBk * chunksPerRow % kThreads == 0, "tile load split");
};

__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ i16x4 lds_read_tr(const uint16_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((ISPA_LDS i16x4*)(p));
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

template <int D>
__global__ __launch_bounds__(kThreads) void attn_chunk_kernel(AttnArgs a, int q_tiles) {
  using C = Cfg<D>;
  __shared__ __attribute__((aligned(16))) uint16_t smem[2 * (C::kTile + C::vTile)];

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

  // ---- global -> register -> LDS staging ------------------------------------------
  u32x4 kreg[C::chunksPerThread], vreg[C::chunksPerThread];
  auto gload = [&](int t) {
    int64_t key0;
    int nv;
    tile_of(a.r, tb1, tb2, t, key0, nv);
#pragma unroll
    for (int c = 0; c < C::chunksPerThread; ++c) {
      const int idx = tid + c * kThreads;
      const int row = idx / C::chunksPerRow;
      const int col = (idx % C::chunksPerRow) * 8;
      if (row < nv) {
        const int64_t off = (key0 + row) * ld + hoff + col;
        kreg[c] = *(const u32x4*)(a.k + off);
        vreg[c] = *(const u32x4*)(a.v + off);
      } else {
        kreg[c] = u32x4{0, 0, 0, 0};
        vreg[c] = u32x4{0, 0, 0, 0};
      }
    }
  };
  auto sstore = [&](int buf) {
    uint16_t* ks = smem + buf * (C::kTile + C::vTile);
    uint16_t* vs = ks + C::kTile;
#pragma unroll
    for (int c = 0; c < C::chunksPerThread; ++c) {
      const int idx = tid + c * kThreads;
      const int row = idx / C::chunksPerRow;
      const int col = (idx % C::chunksPerRow) * 8;
      *(u32x4*)(ks + row * C::kStride + col) = kreg[c];
      *(u32x4*)(vs + row * C::vStride + col) = vreg[c];
    }
  };

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

  if (n_tiles > 0) {
    gload(0);
    sstore(0);
  }
  __syncthreads();

  for (int t = 0; t < n_tiles; ++t) {
    const int buf = t & 1;
    if (dual && t == n_tiles_local) finish(a.out_local, a.lse_local);
    int64_t key0;
    int nv;
    tile_of(a.r, tb1, tb2, t, key0, nv);
    if (t + 1 < n_tiles) gload(t + 1);

    const uint16_t* ks = smem + buf * (C::kTile + C::vTile);
    const uint16_t* vs = ks + C::kTile;

    // S^T = K . Q^T for two 32-key blocks
    f32x16 s[2];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      s[b] = f32x16{};
      const uint16_t* kp = ks + (32 * b + ql) * C::kStride + 8 * hh;
#pragma unroll
      for (int kk = 0; kk < C::kSlices; ++kk) {
        const bf16x8 kf = *(const bf16x8*)(kp + 16 * kk);
        s[b] = mfma32(kf, qf[kk], s[b]);
      }
    }

    // mask keys beyond the end of a range (only the last tile of each range)
    if (nv < kBk) {
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = 32 * b + 8 * (r >> 2) + 4 * hh + (r & 3);
          if (key >= nv) s[b][r] = -INFINITY;
        }
    }

    // online softmax
    float tmax = s[0][0];
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) tmax = fmaxf(tmax, s[b][r]);
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
    const float m_new = fmaxf(m_run, tmax);
    const float alpha = exp2_hw((m_run - m_new) * a.scale_log2);
    const float mc = m_new * a.scale_log2;
    float psum = 0.f;
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = exp2_hw(fmaf(s[b][r], a.scale_log2, -mc));
        s[b][r] = p;
        psum += p;
      }
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int db = 0; db < C::dBlocks; ++db) acc[db] *= alpha;

    // O^T += V^T . P^T over four 16-key slices
    const int g = lane >> 4;
    const int sl = lane & 15;
#pragma unroll
    for (int b = 0; b < 2; ++b) {
#pragma unroll
      for (int t2 = 0; t2 < 2; ++t2) {
        bf16x8 pf;
#pragma unroll
        for (int e = 0; e < 8; ++e) pf[e] = (__bf16)s[b][8 * t2 + e];
        const int slice = 2 * b + t2;
        const uint16_t* vp0 = vs + (16 * slice + 4 * (g >> 1) + (sl >> 2)) * C::vStride +
                              16 * (g & 1) + 4 * (sl & 3);
        const uint16_t* vp1 = vp0 + 8 * C::vStride;
#pragma unroll
        for (int db = 0; db < C::dBlocks; ++db) {
          const i16x4 v0 = lds_read_tr(vp0 + 32 * db);
          const i16x4 v1 = lds_read_tr(vp1 + 32 * db);
          const bf16x8 vf = __builtin_bit_cast(
              bf16x8, __builtin_shufflevector(v0, v1, 0, 1, 2, 3, 4, 5, 6, 7));
          acc[db] = mfma32(vf, pf, acc[db]);
        }
      }
    }

    if (t + 1 < n_tiles) sstore(buf ^ 1);
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
