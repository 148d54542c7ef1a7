// Warmup statistics of layer absorption for gfx950 (CDNA4).
//
// Operation (arXiv 2607.00712, Sec. 3.2): the closed-form modulation only
// needs A_loc^T A_loc and A_loc^T R summed over the warmup rows, where
// R = (A_full - A_loc) W is the full-minus-local output discrepancy.
//
// discrepancy_kernel (HBM-bound, one pass over the rows):
//   R = bf16_rne(fp32(y_full) - fp32(y_local)), s += sum R^2 (fp64 total),
//   and X = bf16_rne(x) when x arrives in fp32. When x is the very same buffer
//   as y_local (the attention output itself, the pre-projection reading) the
//   y_local values already loaded are reused for X.
//   8 elements per thread per step (all loads issued before use), a
//   grid-stride loop over 2 workgroups per CU. Each step's 8 squares are
//   summed in fp32 and added to a per-thread fp64 total; each workgroup leaves
//   its fp64 partial in the caller's workspace, and the Gram kernel that
//   follows on the stream adds the partials to s in workgroup order, so s does
//   not depend on the order in which workgroups run.
//
// gram_kernel (bf16 MFMA 32x32x16, fp32 accumulation):
//   G += X^T X on the lower block triangle of 128x128 tiles, C += X^T R.
//   The contraction runs over rows, the slow (strided) dimension of both
//   operands: row-major stages of 32 rows go HBM -> LDS by buffer loads and both
//   MFMA operands are read with the LDS transpose read (ds_read_b64_tr_b16), 4
//   consecutive rows of one column per lane. Each wave owns a 32 x 64 piece of
//   the tile. When there are fewer tiles than CUs the rows are split in two
//   inside one workgroup of 16 waves (8 per half); the second half's partial
//   tile goes through LDS to the first half, which adds it to its own and then
//   to G or C, so every sum is taken in a fixed order.
#include "ispa_internal.h"

namespace ispa {
namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ uint16_t f2bf_rne(float f) {
  // round-to-nearest-even; NaN stays a quiet NaN
  uint32_t u = __builtin_bit_cast(uint32_t, f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
__device__ __forceinline__ float bf2f(uint16_t b) { return __builtin_bit_cast(float, (uint32_t)b << 16); }

template <int YT>  // element type of y: 0 bf16, 1 f32
__device__ __forceinline__ void load4(const void* p, int64_t i, float v[4]) {
  if (YT == ISPA_DTYPE_F32) {
    const f32x4 t = *(const f32x4*)((const float*)p + i);
    v[0] = t[0]; v[1] = t[1]; v[2] = t[2]; v[3] = t[3];
  } else {
    const u32x2 t = *(const u32x2*)((const uint16_t*)p + i);
    v[0] = bf2f((uint16_t)(t[0] & 0xffff)); v[1] = bf2f((uint16_t)(t[0] >> 16));
    v[2] = bf2f((uint16_t)(t[1] & 0xffff)); v[3] = bf2f((uint16_t)(t[1] >> 16));
  }
}
template <int YT>
__device__ __forceinline__ float load1(const void* p, int64_t i) {
  return YT == ISPA_DTYPE_F32 ? ((const float*)p)[i] : bf2f(((const uint16_t*)p)[i]);
}

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// R and ||R||^2 over n = rows * d_out elements (flat, row-major contiguous);
// X conversion over rows * d_in elements when requested.
template <int YT>
__global__ __launch_bounds__(kThreads) void discrepancy_kernel(
    const void* y_full, const void* y_local, int64_t n_r, uint16_t* r_out, const float* x_f32,
    int64_t n_x, uint16_t* x_out, int x_from_y_local, double* sq_part) {
  __shared__ double red[kThreads / 64];
  const int64_t stride = (int64_t)gridDim.x * kThreads * 8;
  double part = 0.0;
  const int64_t n_r8 = n_r & ~(int64_t)7;
  // 8 elements per thread and step: the four loads are in flight together
  for (int64_t i = ((int64_t)blockIdx.x * kThreads + threadIdx.x) * 8; i < n_r8; i += stride) {
    float f[8], l[8];
    load4<YT>(y_full, i, f);
    load4<YT>(y_full, i + 4, f + 4);
    load4<YT>(y_local, i, l);
    load4<YT>(y_local, i + 4, l + 4);
    uint16_t r[8];
    float step = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      r[j] = f2bf_rne(f[j] - l[j]);
      const float rv = bf2f(r[j]);
      step = fmaf(rv, rv, step);
    }
    part += (double)step;
    u32x4 rw;
#pragma unroll
    for (int j = 0; j < 4; ++j) rw[j] = (uint32_t)r[2 * j] | ((uint32_t)r[2 * j + 1] << 16);
    *(u32x4*)(r_out + i) = rw;
    if (x_from_y_local) {
      u32x4 xw;
#pragma unroll
      for (int j = 0; j < 4; ++j) xw[j] = (uint32_t)f2bf_rne(l[2 * j]) | ((uint32_t)f2bf_rne(l[2 * j + 1]) << 16);
      *(u32x4*)(x_out + i) = xw;
    }
  }
  // ragged tail (fewer than 8 elements), handled by the first workgroup
  if (blockIdx.x == 0 && threadIdx.x < (int)(n_r - n_r8)) {
    const int64_t i = n_r8 + threadIdx.x;
    const float l = load1<YT>(y_local, i);
    const uint16_t r = f2bf_rne(load1<YT>(y_full, i) - l);
    r_out[i] = r;
    const float rv = bf2f(r);
    part += (double)rv * (double)rv;
    if (x_from_y_local) x_out[i] = f2bf_rne(l);
  }
  // separate fp32 -> bf16 conversion of x when it is its own buffer
  if (x_f32 != nullptr && !x_from_y_local) {
    const int64_t n_x4 = n_x & ~(int64_t)3;
    for (int64_t i = ((int64_t)blockIdx.x * kThreads + threadIdx.x) * 4; i < n_x4; i += stride / 2) {
      const f32x4 t = *(const f32x4*)(x_f32 + i);
      *(u32x2*)(x_out + i) = u32x2{(uint32_t)f2bf_rne(t[0]) | ((uint32_t)f2bf_rne(t[1]) << 16),
                                   (uint32_t)f2bf_rne(t[2]) | ((uint32_t)f2bf_rne(t[3]) << 16)};
    }
    if (blockIdx.x == 0 && threadIdx.x < (int)(n_x - n_x4)) {
      const int64_t i = n_x4 + threadIdx.x;
      x_out[i] = f2bf_rne(x_f32[i]);
    }
  }
  double d = wave_sum(part);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = d;
  __syncthreads();
  if (threadIdx.x == 0) {
    double t = 0;
#pragma unroll
    for (int w = 0; w < kThreads / 64; ++w) t += red[w];
    sq_part[blockIdx.x] = t;
  }
}

// ---------------------------------------------------------------- Gram
// Output tiles of 128 x 128 on the lower block triangle of G and all of C,
// one workgroup of 8 waves per tile (two waves per SIMD), wave w owning rows
// 32 (w / 2) .. +31 and columns 64 (w % 2) .. +63 (1 x 2 accumulator blocks of
// 32 x 32). Rows are staged 32 at a time HBM -> LDS by buffer loads (no register
// staging) into a ring of 4 stage buffers, 3 stages ahead of the MFMAs; a stage
// holds the 32 rows of the tile's 128 X columns (A side) and of its 128 X or R
// columns (B side) as 256-byte rows (16 KB). Both MFMA operands need 8
// consecutive rows of one column per lane, which the LDS transpose read
// delivers (two reads of 4 rows); the 16-byte chunk index of each row is
// XOR-swizzled with 4 (row mod 4) ^ 2 (row/4 mod 2) so that the 32 lanes of a
// transpose read hit 16 distinct chunk positions. The buffer descriptor of a
// stage ends at the split's last row, so rows past it read as zero; columns
// past d of a ragged last tile read neighbouring data that only reaches output
// rows/columns >= d, which are never stored. When the tiles number fewer than
// the 256 CUs, the rows are split in two inside a workgroup of 16 waves, each
// half with its own ring (16 waves per CU hide each other's latencies as two
// 8-wave workgroups would), and the halves are added through LDS in a fixed
// order; every tile is then added to G or C with plain read-modify-writes. Measured against 256 x 256 tiles of 8
// waves of 64 x 128 (row splits and atomics to fill the chip): 0.081 vs 0.098 ms
// per 4680-row chunk at d = 1536, 0.514 vs 0.531 ms at d = 5120.
constexpr int kGK = 32;                        // rows per stage
constexpr int kGRing = 4;                      // stage buffers
constexpr int kHalfBytes = kGK * 256;          // one 32 x 128 side (bf16)
constexpr int kG2Threads = 512;
constexpr int kG2Waves = kG2Threads / 64;
constexpr int kG2T = 128;                                    // output tile (rows and columns)
constexpr int kG2Stage = 2 * kHalfBytes;                     // A side + B side
constexpr int kG2Loads = kG2Stage / (kG2Threads * 16);       // direct loads per thread per stage
__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ int gswz(int row) { return (4 * (row & 3)) ^ (2 * ((row >> 2) & 1)); }
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int nbytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, nbytes, 0x00020000);
}
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(ISPA_LDS const void*)p;
}

// Wait until at most N vector memory operations of this wave are outstanding.
template <int N>
__device__ __forceinline__ void vm_wait() {
  static_assert(N >= 0 && N <= 63, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"i"(N) : "memory");
}

struct GramArgs {
  const uint16_t* x;  // [rows, d_in]
  const uint16_t* r;  // [rows, d_out]
  float* G;           // [d_in, d_in]
  float* C;           // [d_in, d_out]
  int64_t rows;
  int d_in, d_out;
  int tiles_in, tiles_out;  // output tiles along d_in / d_out
  int n_g_tiles;            // lower block triangle of G
  int n_tiles;              // G tiles + C tiles
  int64_t rows_per_split;   // rows of each half of a split workgroup (multiple of kGK)
  const double* sq_part;    // norm partials of the discrepancy kernel, added to *sq_norm by workgroup 0
  double* sq_norm;
  int n_sq_part;
};

// Transpose-read addresses of one side for this lane, stage buffer 0, k-slice
// 0: [blk][h] for column block blk0 + blk (32 columns of a 128-column half) and
// row half h (rows +4). The swizzle of a row depends only on (row mod 4,
// row/4 mod 2), i.e. on the lane and h, so k-slices and stage buffers are pure
// immediate offsets.
template <int NB>
struct SideAddr {
  uint32_t a[NB][2];
};
template <int NB>
__device__ __forceinline__ void side_addr(SideAddr<NB>& s, uint32_t half_base, int blk0, int lane) {
  const int g = lane >> 4, sl = lane & 15;
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int row = 8 * (g >> 1) + 4 * h + (sl >> 2);
      const int chunk = 4 * (blk0 + b) + 2 * (g & 1) + ((sl & 3) >> 1);
      s.a[b][h] = half_base + row * 256 + ((chunk ^ gswz(row)) << 4) + ((sl & 1) << 3);
    }
}

struct GramTile {
  const uint16_t* bsrc;
  int64_t bld;
  int64_t r_begin, r_end;
  int row0, col0, steps, wave, lane;
};

// Output tile k of one split in panel-group order: row panels (X columns) are
// taken kGroup at a time; within a group the G tiles of the lower block
// triangle come column by column, then the C tiles column by column, each
// column holding the group's rows. Returns true for a G tile (ti, tj: row and
// column panel), false for a C tile.
constexpr int kGroup = 4;
__device__ __forceinline__ bool gram_tile_of(int k, int tiles_in, int tiles_out, int& ti, int& tj) {
  int r0 = 0, gm = 0, n_g = 0;
  for (;; r0 += kGroup) {
    gm = min(kGroup, tiles_in - r0);
    n_g = r0 * gm + gm * (gm + 1) / 2;
    const int n = n_g + tiles_out * gm;
    if (k < n || r0 + gm >= tiles_in) break;
    k -= n;
  }
  if (k < r0 * gm) {  // full columns left of the group's diagonal block
    tj = k / gm;
    ti = r0 + k % gm;
    return true;
  }
  if (k < n_g) {  // the diagonal block's lower triangle: column c holds rows c .. r0 + gm - 1
    k -= r0 * gm;
    tj = r0;
    while (k >= r0 + gm - tj) {
      k -= r0 + gm - tj;
      ++tj;
    }
    ti = tj + k;
    return true;
  }
  k -= n_g;
  tj = k / gm;
  ti = r0 + k % gm;
  return false;
}

// Direct loads of one 32-row x 128-column side: load q of wave w covers 16-byte
// slot (q * 8 + w) * 64 + lane, row = (slot / 16) % 32, stored chunk = slot % 16.
__device__ __forceinline__ void stage_half(const uint16_t* src, int64_t ld, int64_t row0, int64_t row_end, int col0,
                                           char* dst, int wave, int lane) {
  int64_t nrec = ((row_end - row0) * ld - col0) * 2;
  if (nrec < 0) nrec = 0;
  if (nrec > 0x7fffffff) nrec = 0x7fffffff;
  const __amdgpu_buffer_rsrc_t rs = make_rsrc(src + row0 * ld + col0, (int)nrec);
#pragma unroll
  for (int q = 0; q < kHalfBytes / (kG2Threads * 16); ++q) {
    const int slot = (q * kG2Waves + wave) * 64 + lane;
    const int row = (slot >> 4) & 31;
    const int c = (slot & 15) ^ gswz(row);
    const int voff = (int)((row * ld + c * 8) * 2);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (ISPA_LDS void*)(dst + (q * kG2Waves + wave) * 1024), 16, voff, 0,
                                             0, 0);
  }
}

// The 8 transpose reads (2 A blocks, 2 B blocks, 2 row halves each) of one
// 16-row slice and the wait for them.
template <int IMM, int NA>
__device__ __forceinline__ void gram2_issue(const SideAddr<NA>& A, const SideAddr<2>& B, u32x2 (&ra)[NA][2],
                                            u32x2 (&rb)[2][2]) {
#pragma unroll
  for (int b = 0; b < NA; ++b)
#pragma unroll
    for (int h = 0; h < 2; ++h)
      asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(ra[b][h]) : "v"(A.a[b][h]), "i"(IMM));
#pragma unroll
  for (int b = 0; b < 2; ++b)
#pragma unroll
    for (int h = 0; h < 2; ++h)
      asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(rb[b][h]) : "v"(B.a[b][h]), "i"(IMM));
}
template <int N>
__device__ __forceinline__ void gram2_wait(u32x2 (&ra)[1][2], u32x2 (&rb)[2][2], bf16x8* af, bf16x8* bf) {
  static_assert(N >= 0 && N <= 15, "lgkmcnt range");
  asm volatile("s_waitcnt lgkmcnt(%6)"
               : "+v"(ra[0][0]), "+v"(ra[0][1]), "+v"(rb[0][0]), "+v"(rb[0][1]), "+v"(rb[1][0]), "+v"(rb[1][1])
               : "i"(N));
  af[0] = __builtin_bit_cast(bf16x8, u32x4{ra[0][0][0], ra[0][0][1], ra[0][1][0], ra[0][1][1]});
#pragma unroll
  for (int b = 0; b < 2; ++b)
    bf[b] = __builtin_bit_cast(bf16x8, u32x4{rb[b][0][0], rb[b][0][1], rb[b][1][0], rb[b][1][1]});
}

__device__ __forceinline__ void stage2_load(const GramArgs& a, const GramTile& t, char* smem, int s) {
  const int64_t rr = t.r_begin + (int64_t)s * kGK;
  char* d = smem + (s % kGRing) * kG2Stage;
  stage_half(a.x, a.d_in, rr, t.r_end, t.row0, d, t.wave, t.lane);
  stage_half(t.bsrc, t.bld, rr, t.r_end, t.col0, d + kHalfBytes, t.wave, t.lane);
}

// Stage s from ring buffer BUF = s % 4: loads of stage s + 3, the 8 MFMAs of
// this wave (the second slice's reads in flight during the first slice's
// MFMAs), then wait for stage s + 1 and synchronise.
template <int BUF>
__device__ __forceinline__ void gram2_stage(const GramArgs& a, const GramTile& t, char* smem, const SideAddr<1>& A,
                                            const SideAddr<2>& B, f32x16 (&acc)[2], int s) {
  constexpr int kOff = BUF * kG2Stage;
  if (s + 3 < t.steps) stage2_load(a, t, smem, s + 3);
  u32x2 ra[1][2], rb[2][2];
  bf16x8 af[1], bf[2];
  gram2_issue<kOff, 1>(A, B, ra, rb);
  gram2_wait<0>(ra, rb, af, bf);
  gram2_issue<kOff + 16 * 256, 1>(A, B, ra, rb);
#pragma unroll
  for (int j = 0; j < 2; ++j) acc[j] = mfma32(af[0], bf[j], acc[j]);
  gram2_wait<0>(ra, rb, af, bf);
#pragma unroll
  for (int j = 0; j < 2; ++j) acc[j] = mfma32(af[0], bf[j], acc[j]);
  const int younger = t.steps - (s + 2);
  if (younger >= 2) {
    vm_wait<2 * kG2Loads>();
  } else if (younger == 1) {
    vm_wait<kG2Loads>();
  } else {
    vm_wait<0>();
  }
  __builtin_amdgcn_s_barrier();
}

// The norm partials of the discrepancy kernel that ran before on the stream,
// added to s in workgroup order (one wave: lane i takes partials i, i + 64,
// ..., then a fixed shuffle tree).
__device__ void add_sq_parts(const GramArgs& a) {
  double sq = 0.0;
  for (int b = threadIdx.x; b < a.n_sq_part; b += 64) sq += a.sq_part[b];
  sq = wave_sum(sq);
  if (threadIdx.x == 0) *a.sq_norm += sq;
}

// The same on its own, beside the hand-scheduled Gram kernel (one wave).
__global__ __launch_bounds__(64) void sq_norm_kernel(GramArgs a) { add_sq_parts(a); }

// After a hand-scheduled Gram launch that split tiles into row pieces: tile
// n_whole + q (256 x 256, the panel-group order) += the sums of pieces 1 ..
// pieces - 1 in scratch slots (piece - 1) n_split + q, in piece order; piece 0
// has already added its own, so every element is summed in a fixed order. 64
// workgroups per tile, 4 rows each; the first wave of the first one also adds
// the norm partials (as sq_norm_kernel does without a fixup).
__global__ __launch_bounds__(256) void gram_fixup_kernel(GramArgs a, const float* ws, int n_whole, int n_split,
                                                         int pieces, int tiles_in, int tiles_out) {
  if (blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x < 64) add_sq_parts(a);
  float *G = a.G, *C = a.C;
  const int d_in = a.d_in, d_out = a.d_out;
  const int q = blockIdx.y;
  int ti, tj;
  const bool is_g = gram_tile_of(n_whole + q, tiles_in, tiles_out, ti, tj);
  float* out = is_g ? G : C;
  const int ld = is_g ? d_in : d_out;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6), col = (threadIdx.x & 63) * 4;
  f32x4* o = (f32x4*)(out + (int64_t)(256 * ti + row) * ld + 256 * tj + col);
  // the pieces after the first, in piece order (slot (piece - 1) n_split + q)
  f32x4 v = *o;
  for (int p = 1; p < pieces; ++p) v = v + *(const f32x4*)(ws + ((int64_t)(p - 1) * n_split + q) * 65536 + row * 256 + col);
  *o = v;
}

// SPLIT = 2: 16 waves, waves 8..15 take the second half of the rows with
// their own ring, and their partial tile reaches waves 0..7 through LDS.
template <int SPLIT>
__global__ __launch_bounds__(kG2Threads * SPLIT) __attribute__((amdgpu_waves_per_eu(2 * SPLIT))) void gram_kernel(
    GramArgs a) {
  __shared__ __attribute__((aligned(1024))) char smem_all[SPLIT * kGRing * kG2Stage];
  if (blockIdx.x == 0 && threadIdx.x < 64) add_sq_parts(a);
  // The work list (tiles in panel-group order) is cut into 8 contiguous
  // ranges, one per XCD (workgroups are dealt to the XCDs round robin), so
  // that the workgroups resident on one XCD at a time work on few distinct
  // X / R panels and share them through that XCD's L2.
  const int n_items = a.n_tiles;
  const int per_xcd = (n_items + 7) / 8;
  const int item = (int)(blockIdx.x % 8) * per_xcd + (int)(blockIdx.x / 8);
  if (item >= n_items) return;
  const int half = SPLIT > 1 ? (int)(threadIdx.x / kG2Threads) : 0;
  const int tid = (int)threadIdx.x - half * kG2Threads;
  char* smem = smem_all + half * kGRing * kG2Stage;
  GramTile t;
  int ti, tj;
  const bool is_g = gram_tile_of(item, a.tiles_in, a.tiles_out, ti, tj);
  float* out;
  int out_ld, out_cols;
  if (is_g) {
    t.bsrc = a.x; t.bld = a.d_in; out = a.G; out_ld = a.d_in; out_cols = a.d_in;
  } else {
    t.bsrc = a.r; t.bld = a.d_out; out = a.C; out_ld = a.d_out; out_cols = a.d_out;
  }
  t.row0 = ti * kG2T;
  t.col0 = tj * kG2T;
  t.r_begin = (int64_t)half * a.rows_per_split;
  t.r_end = t.r_begin + a.rows_per_split;
  if (t.r_end > a.rows) t.r_end = a.rows;
  t.lane = tid & 63;
  t.wave = tid >> 6;
  // both halves run the same number of stages (they share the barriers);
  // stages past a half's last row read zeros
  t.steps = (int)((a.rows_per_split + kGK - 1) / kGK);
  const int wr = t.wave >> 1;  // output rows 32 wr .. +31: A block wr
  const int wc = t.wave & 1;   // output cols 64 wc .. +63: B blocks 2 wc, +1

  const uint32_t lds0 = lds_addr(smem);
  SideAddr<1> A;
  SideAddr<2> B;
  side_addr<1>(A, lds0, wr, t.lane);
  side_addr<2>(B, lds0 + kHalfBytes, 2 * wc, t.lane);

  f32x16 acc[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) acc[j] = f32x16{};

  for (int s = 0; s < 3 && s < t.steps; ++s) stage2_load(a, t, smem, s);
  if (t.steps >= 3) {
    vm_wait<2 * kG2Loads>();
  } else if (t.steps == 2) {
    vm_wait<kG2Loads>();
  } else {
    vm_wait<0>();
  }
  __builtin_amdgcn_s_barrier();  // stage 0 has landed (vmcnt above)
  for (int s = 0; s < t.steps; s += kGRing) {
    gram2_stage<0>(a, t, smem, A, B, acc, s);
    if (s + 1 < t.steps) gram2_stage<1>(a, t, smem, A, B, acc, s + 1);
    if (s + 2 < t.steps) gram2_stage<2>(a, t, smem, A, B, acc, s + 2);
    if (s + 3 < t.steps) gram2_stage<3>(a, t, smem, A, B, acc, s + 3);
  }
  if constexpr (SPLIT > 1) {
    // the second half's tile through its (now idle) ring, 16 bytes per lane
    // and store: [k][tid] for the 8 f32x4 pieces k of a thread's 32 values
    f32x4* xch = (f32x4*)(smem_all + kGRing * kG2Stage);
    __syncthreads();
    if (half == 1) {
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          xch[(4 * j + i) * kG2Threads + tid] = f32x4{acc[j][4 * i], acc[j][4 * i + 1], acc[j][4 * i + 2],
                                                      acc[j][4 * i + 3]};
    }
    __syncthreads();
    if (half == 1) return;
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const f32x4 o = xch[(4 * j + i) * kG2Threads + tid];
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[j][4 * i + e] += o[e];
      }
  }
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int orow = t.row0 + 32 * wr + 8 * (r >> 2) + 4 * (t.lane >> 5) + (r & 3);
      const int ocol = t.col0 + 64 * wc + 32 * j + (t.lane & 31);
      if (orow < a.d_in && ocol < out_cols) out[(int64_t)orow * out_ld + ocol] += acc[j][r];
    }
}

__global__ void zero_kernel(uint32_t* p, int64_t n_words) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_words;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0u;
}

}  // namespace

hipError_t launch_zero(void* p, size_t bytes, hipStream_t stream) {
  const int64_t words = (int64_t)(bytes / 4);
  if (words == 0) return hipSuccess;
  int grid = (int)((words + 255) / 256);
  if (grid > 4096) grid = 4096;
  hipLaunchKernelGGL(zero_kernel, dim3(grid), dim3(256), 0, stream, (uint32_t*)p, words);
  return hipGetLastError();
}

int discrepancy_grid(int64_t rows, int d_in, int d_out) {
  const int64_t n_r = rows * d_out;
  const int64_t n_x = rows * d_in;
  const int64_t n_max = n_r > n_x ? n_r : n_x;
  int64_t grid = (n_max / 8 + kThreads - 1) / kThreads;
  // 2 workgroups per CU, grid-stride beyond (measured: 256-512 workgroups
  // best at the 1.3B chunk)
  if (grid > kDiscMaxGrid) grid = kDiscMaxGrid;
  if (grid < 1) grid = 1;
  return (int)grid;
}

hipError_t launch_discrepancy(const void* x, int x_dtype, const void* y_full, const void* y_local,
                              int y_dtype, int64_t rows, int d_in, int d_out, uint16_t* x_bf16,
                              uint16_t* r_bf16, double* sq_part, hipStream_t stream) {
  const int64_t n_r = rows * d_out;
  const int64_t n_x = rows * d_in;
  const bool x_from_y = x_dtype == ISPA_DTYPE_F32 && y_dtype == ISPA_DTYPE_F32 && x == y_local &&
                        d_in == d_out;
  const float* x_f32 = x_dtype == ISPA_DTYPE_F32 ? (const float*)x : nullptr;
  const int grid = discrepancy_grid(rows, d_in, d_out);
  if (y_dtype == ISPA_DTYPE_F32) {
    hipLaunchKernelGGL(discrepancy_kernel<ISPA_DTYPE_F32>, dim3((unsigned)grid), dim3(kThreads), 0,
                       stream, y_full, y_local, n_r, r_bf16, x_f32, n_x, x_bf16, (int)x_from_y,
                       sq_part);
  } else {
    hipLaunchKernelGGL(discrepancy_kernel<ISPA_DTYPE_BF16>, dim3((unsigned)grid), dim3(kThreads), 0,
                       stream, y_full, y_local, n_r, r_bf16, x_f32, n_x, x_bf16, (int)x_from_y,
                       sq_part);
  }
  return hipGetLastError();
}

int gram_tiles(int d_in, int d_out) {
  const int ti = (d_in + kG2T - 1) / kG2T, to = (d_out + kG2T - 1) / kG2T;
  return ti * (ti + 1) / 2 + ti * to;
}

hipError_t launch_gram(const uint16_t* x, const uint16_t* r, int64_t rows, int d_in, int d_out,
                       float* G, float* C, const double* sq_part, int n_sq_part, double* sq_norm,
                       float* scratch, size_t scratch_bytes, hipStream_t stream) {
  if (rows <= 0) return hipSuccess;
  GramArgs a;
  a.x = x; a.r = r; a.G = G; a.C = C; a.rows = rows; a.d_in = d_in; a.d_out = d_out;
  a.sq_part = sq_part;
  a.n_sq_part = n_sq_part;
  a.sq_norm = sq_norm;
  GramFastPlan plan;
  if (gram_fast_plan(rows, d_in, d_out, scratch != nullptr ? scratch_bytes : 0, &plan)) {
    hipError_t e = launch_gram_fast(x, r, rows, d_in, d_out, G, C, scratch, plan, stream);
    if (e != hipSuccess) return e;
    if (plan.n_split == 0) {
      hipLaunchKernelGGL(sq_norm_kernel, dim3(1), dim3(64), 0, stream, a);
    } else {
      hipLaunchKernelGGL(gram_fixup_kernel, dim3(64, plan.n_split), dim3(256), 0, stream, a, scratch, plan.n_whole,
                         plan.n_split, 1 << plan.log_pieces, d_in / 256, d_out / 256);
    }
    return hipGetLastError();
  }
  a.tiles_in = (d_in + kG2T - 1) / kG2T;
  a.tiles_out = (d_out + kG2T - 1) / kG2T;
  a.n_g_tiles = a.tiles_in * (a.tiles_in + 1) / 2;
  a.n_tiles = a.n_g_tiles + a.tiles_in * a.tiles_out;
  // fewer tiles than CUs: the rows split in two inside each workgroup (each
  // half of at least 8 stages)
  const bool split = a.n_tiles < kGramSplitTiles && rows >= 2 * 8 * kGK;
  int64_t per = split ? (rows + 1) / 2 : rows;
  per = (per + kGK - 1) / kGK * kGK;
  a.rows_per_split = per;
  const dim3 grid((unsigned)(8 * ((a.n_tiles + 7) / 8)));
  if (split) {
    hipLaunchKernelGGL(gram_kernel<2>, grid, dim3(2 * kG2Threads), 0, stream, a);
  } else {
    hipLaunchKernelGGL(gram_kernel<1>, grid, dim3(kG2Threads), 0, stream, a);
  }
  return hipGetLastError();
}

}  // namespace ispa
