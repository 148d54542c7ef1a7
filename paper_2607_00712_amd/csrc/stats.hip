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
//   Vector loads of 4 elements per thread per step, a grid-stride loop sized to
//   the device, wavefront shuffles then one fp64 atomic per workgroup.
//
// gram_kernel (bf16 MFMA 32x32x16, fp32 accumulation):
//   G += X^T X on the lower block triangle of 128x128 tiles, C += X^T R.
//   The contraction runs over rows, which are the slow (strided) dimension of
//   both operands. Row-major tiles of 32 rows x 128 columns are staged in LDS
//   and both MFMA operands are read with the LDS transpose read
//   (ds_read_b64_tr_b16), which returns 4 consecutive rows of one column per
//   lane. A workgroup (4 waves, 2x2 of 64x64) owns one output tile; the rows
//   are split over several workgroups when there are too few tiles to fill the
//   256 CUs, and partial sums are added with fp32 atomics.
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
    int64_t n_x, uint16_t* x_out, int x_from_y_local, double* sq_norm) {
  __shared__ double red[kThreads / 64];
  const int64_t stride = (int64_t)gridDim.x * kThreads * 4;
  float part = 0.f;
  const int64_t n_r4 = n_r & ~(int64_t)3;
  for (int64_t i = ((int64_t)blockIdx.x * kThreads + threadIdx.x) * 4; i < n_r4; i += stride) {
    float f[4], l[4];
    load4<YT>(y_full, i, f);
    load4<YT>(y_local, i, l);
    uint16_t r[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      r[j] = f2bf_rne(f[j] - l[j]);
      const float rv = bf2f(r[j]);
      part = fmaf(rv, rv, part);
    }
    *(u32x2*)(r_out + i) = u32x2{(uint32_t)r[0] | ((uint32_t)r[1] << 16),
                                 (uint32_t)r[2] | ((uint32_t)r[3] << 16)};
    if (x_from_y_local) {
      *(u32x2*)(x_out + i) = u32x2{(uint32_t)f2bf_rne(l[0]) | ((uint32_t)f2bf_rne(l[1]) << 16),
                                   (uint32_t)f2bf_rne(l[2]) | ((uint32_t)f2bf_rne(l[3]) << 16)};
    }
  }
  // ragged tail (fewer than 4 elements), handled by the first workgroup
  if (blockIdx.x == 0 && threadIdx.x < (int)(n_r - n_r4)) {
    const int64_t i = n_r4 + threadIdx.x;
    const float l = load1<YT>(y_local, i);
    const uint16_t r = f2bf_rne(load1<YT>(y_full, i) - l);
    r_out[i] = r;
    const float rv = bf2f(r);
    part = fmaf(rv, rv, part);
    if (x_from_y_local) x_out[i] = f2bf_rne(l);
  }
  // separate fp32 -> bf16 conversion of x when it is its own buffer
  if (x_f32 != nullptr && !x_from_y_local) {
    const int64_t n_x4 = n_x & ~(int64_t)3;
    for (int64_t i = ((int64_t)blockIdx.x * kThreads + threadIdx.x) * 4; i < n_x4; i += stride) {
      const f32x4 t = *(const f32x4*)(x_f32 + i);
      *(u32x2*)(x_out + i) = u32x2{(uint32_t)f2bf_rne(t[0]) | ((uint32_t)f2bf_rne(t[1]) << 16),
                                   (uint32_t)f2bf_rne(t[2]) | ((uint32_t)f2bf_rne(t[3]) << 16)};
    }
    if (blockIdx.x == 0 && threadIdx.x < (int)(n_x - n_x4)) {
      const int64_t i = n_x4 + threadIdx.x;
      x_out[i] = f2bf_rne(x_f32[i]);
    }
  }
  double d = wave_sum((double)part);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = d;
  __syncthreads();
  if (threadIdx.x == 0) {
    double t = 0;
#pragma unroll
    for (int w = 0; w < kThreads / 64; ++w) t += red[w];
    if (t != 0.0) atomicAdd(sq_norm, t);
  }
}

// ---------------------------------------------------------------- Gram
constexpr int kTile = 128;   // output tile (rows and columns)
constexpr int kRows = 32;    // rows staged per step
constexpr int kLds = kTile + 16;  // LDS row stride (elements) for the tr reads

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ i16x4 lds_read_tr(const uint16_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((ISPA_LDS i16x4*)(p));
}

// Operand for rows [16*ks, 16*ks+16) and 32 columns starting at col0 of a
// row-major LDS tile: lane l gets column col0 + l%32, rows 16ks + 8(l/32) + 0..7.
__device__ __forceinline__ bf16x8 tr_operand(const uint16_t* tile, int ks, int col0, int lane) {
  const int g = lane >> 4, sl = lane & 15;
  const uint16_t* p = tile + (16 * ks + 8 * (g >> 1) + (sl >> 2)) * kLds + col0 + 16 * (g & 1) + 4 * (sl & 3);
  const i16x4 v0 = lds_read_tr(p);
  const i16x4 v1 = lds_read_tr(p + 4 * kLds);
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(v0, v1, 0, 1, 2, 3, 4, 5, 6, 7));
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
  int splits;               // row splits
  int64_t rows_per_split;   // multiple of kRows
};

__global__ __launch_bounds__(kThreads) void gram_kernel(GramArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t sA[2][kRows * kLds];
  __shared__ __attribute__((aligned(16))) uint16_t sB[2][kRows * kLds];

  const int tile = blockIdx.x % a.n_tiles;
  const int split = blockIdx.x / a.n_tiles;
  int ti, tj;
  const uint16_t* bsrc;
  int bld;
  float* out;
  int out_ld, out_cols;
  if (tile < a.n_g_tiles) {
    // lower block triangle: tile = ti (ti + 1) / 2 + tj, tj <= ti
    ti = (int)((sqrtf(8.f * tile + 1.f) - 1.f) * 0.5f);
    while ((ti + 1) * (ti + 2) / 2 <= tile) ++ti;
    while (ti * (ti + 1) / 2 > tile) --ti;
    tj = tile - ti * (ti + 1) / 2;
    bsrc = a.x; bld = a.d_in; out = a.G; out_ld = a.d_in; out_cols = a.d_in;
  } else {
    const int c = tile - a.n_g_tiles;
    ti = c / a.tiles_out;
    tj = c % a.tiles_out;
    bsrc = a.r; bld = a.d_out; out = a.C; out_ld = a.d_out; out_cols = a.d_out;
  }
  const int row0 = ti * kTile;  // output rows = X columns
  const int col0 = tj * kTile;  // output cols = X or R columns
  const int64_t r_begin = (int64_t)split * a.rows_per_split;
  int64_t r_end = r_begin + a.rows_per_split;
  if (r_end > a.rows) r_end = a.rows;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wr = (wave >> 1) * 64;  // wave's output sub-tile
  const int wc = (wave & 1) * 64;

  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x16{};

  // staging: 32 rows x 128 columns of each operand = 512 chunks of 8 bf16,
  // two per thread per operand
  u32x4 ra[2], rb[2];
  auto gload = [&](int64_t r0) {
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int idx = tid + c * kThreads;
      const int rr = idx >> 4;
      const int cc = (idx & 15) * 8;
      const int64_t row = r0 + rr;
      const bool rok = row < r_end;
      ra[c] = (rok && row0 + cc < a.d_in) ? *(const u32x4*)(a.x + row * a.d_in + row0 + cc) : u32x4{0, 0, 0, 0};
      rb[c] = (rok && col0 + cc < out_cols) ? *(const u32x4*)(bsrc + row * bld + col0 + cc) : u32x4{0, 0, 0, 0};
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int idx = tid + c * kThreads;
      const int rr = idx >> 4;
      const int cc = (idx & 15) * 8;
      *(u32x4*)(&sA[buf][rr * kLds + cc]) = ra[c];
      *(u32x4*)(&sB[buf][rr * kLds + cc]) = rb[c];
    }
  };

  const int steps = r_end > r_begin ? (int)((r_end - r_begin + kRows - 1) / kRows) : 0;
  if (steps > 0) {
    gload(r_begin);
    sstore(0);
  }
  __syncthreads();
  for (int s = 0; s < steps; ++s) {
    const int buf = s & 1;
    if (s + 1 < steps) gload(r_begin + (int64_t)(s + 1) * kRows);
#pragma unroll
    for (int ks = 0; ks < kRows / 16; ++ks) {
      bf16x8 af[2], bf[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) af[i] = tr_operand(sA[buf], ks, wr + 32 * i, lane);
#pragma unroll
      for (int j = 0; j < 2; ++j) bf[j] = tr_operand(sB[buf], ks, wc + 32 * j, lane);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = mfma32(af[i], bf[j], acc[i][j]);
    }
    if (s + 1 < steps) sstore(buf ^ 1);
    __syncthreads();
  }

  // accumulate into G / C: lane holds column (lane%32) and rows 8(r/4)+4(lane/32)+r%4
  const bool atomic = a.splits > 1;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int orow = row0 + wr + 32 * i + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        const int ocol = col0 + wc + 32 * j + (lane & 31);
        if (orow < a.d_in && ocol < out_cols) {
          float* p = out + (int64_t)orow * out_ld + ocol;
          if (atomic) {
            atomicAdd(p, acc[i][j][r]);
          } else {
            *p += acc[i][j][r];
          }
        }
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

hipError_t launch_discrepancy(const void* x, int x_dtype, const void* y_full, const void* y_local,
                              int y_dtype, int64_t rows, int d_in, int d_out, uint16_t* x_bf16,
                              uint16_t* r_bf16, double* sq_norm, hipStream_t stream) {
  const int64_t n_r = rows * d_out;
  const int64_t n_x = rows * d_in;
  const bool x_from_y = x_dtype == ISPA_DTYPE_F32 && y_dtype == ISPA_DTYPE_F32 && x == y_local &&
                        d_in == d_out;
  const float* x_f32 = x_dtype == ISPA_DTYPE_F32 ? (const float*)x : nullptr;
  const int64_t n_max = n_r > n_x ? n_r : n_x;
  int64_t grid = (n_max / 4 + kThreads - 1) / kThreads;
  if (grid > 2048) grid = 2048;  // 8 workgroups per CU, grid-stride beyond
  if (grid < 1) grid = 1;
  if (y_dtype == ISPA_DTYPE_F32) {
    hipLaunchKernelGGL(discrepancy_kernel<ISPA_DTYPE_F32>, dim3((unsigned)grid), dim3(kThreads), 0,
                       stream, y_full, y_local, n_r, r_bf16, x_f32, n_x, x_bf16, (int)x_from_y,
                       sq_norm);
  } else {
    hipLaunchKernelGGL(discrepancy_kernel<ISPA_DTYPE_BF16>, dim3((unsigned)grid), dim3(kThreads), 0,
                       stream, y_full, y_local, n_r, r_bf16, x_f32, n_x, x_bf16, (int)x_from_y,
                       sq_norm);
  }
  return hipGetLastError();
}

hipError_t launch_gram(const uint16_t* x, const uint16_t* r, int64_t rows, int d_in, int d_out,
                       float* G, float* C, hipStream_t stream) {
  if (rows <= 0) return hipSuccess;
  GramArgs a;
  a.x = x; a.r = r; a.G = G; a.C = C; a.rows = rows; a.d_in = d_in; a.d_out = d_out;
  a.tiles_in = (d_in + kTile - 1) / kTile;
  a.tiles_out = (d_out + kTile - 1) / kTile;
  a.n_g_tiles = a.tiles_in * (a.tiles_in + 1) / 2;
  a.n_tiles = a.n_g_tiles + a.tiles_in * a.tiles_out;
  // enough workgroups for 2 per CU, but at least 256 rows per split
  int splits = (512 + a.n_tiles - 1) / a.n_tiles;
  const int64_t max_splits = (rows + 255) / 256;
  if (splits > max_splits) splits = (int)max_splits;
  if (splits < 1) splits = 1;
  int64_t per = (rows + splits - 1) / splits;
  per = (per + kRows - 1) / kRows * kRows;
  splits = (int)((rows + per - 1) / per);
  a.splits = splits;
  a.rows_per_split = per;
  hipLaunchKernelGGL(gram_kernel, dim3((unsigned)(a.n_tiles * splits)), dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace ispa
