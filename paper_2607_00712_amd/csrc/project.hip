// Output projection of an L-Layer for gfx950 (CDNA4).
//
// Operation (arXiv 2607.00712, Sec. 3.1 step 3 with Eq. 4): after absorption an
// L-Layer projects its local attention output with the modulated weight,
// Y = A W_new. The weight is taken in the linear-layer layout W_lin = W_new^T
// [d_out, d_in] (the layout ispa_inject_modulation updates with dW^T), so
// Y = A W_lin^T and both operands have the contraction dimension contiguous.
//
// proj_kernel (bf16 MFMA 32x32x16, fp32 accumulation): output tile 128 MB rows
// x TN columns (256 x 256, 256 x 128, or 128 x 128 for the int8 form), 8 waves
// (two per SIMD); wave w owns rows 32 MB (w / 2) .. +32 MB - 1 and columns
// (TN / 2)(w % 2) .. +TN/2 - 1. Stages of 32 k go HBM -> LDS by direct buffer
// loads into a ring of 4 buffers, 3 stages ahead of the MFMAs, one barrier per
// stage. LDS rows are
// 64 bytes (four 16-byte chunks of 8 k); the chunk index is XOR-swizzled with
// (row / 4) mod 4 so that each 16-lane group of an operand read (16
// consecutive rows, one chunk) covers all 64 banks. Rows past n_rows or d_out
// read as zero through the buffer descriptors and are never stored.
//
// The same kernel computes the W8A8 form (Sec. 4 pairs the method with int8
// linear layers): int8 codes of A and W_lin, int8 MFMA 32x32x32 with int32
// accumulation, 64 k per stage so that LDS rows stay 64 bytes, and the
// dequantisation y = (float(acc) * s_a[row]) * s_w[col] in the epilogue.
// quant_rows_kernel produces the codes: one wave per row, symmetric scale
// absmax / 127, codes rint(x / scale) clamped to +-127.
#include "ispa_internal.h"

namespace ispa {
namespace {

constexpr int kPThreads = 512;
constexpr int kPRowBytes = 64;    // bytes of k per row per stage (32 bf16 or 64 int8)
constexpr int kPRing = 4;         // stage buffers

// TN tile columns; MB 32-row accumulator blocks per wave, so tiles of 128 MB rows
template <int TN, int MB>
struct PCfg {
  static constexpr int tm = 128 * MB;            // tile rows (rows of A)
  static constexpr int sideA = tm * kPRowBytes;
  static constexpr int sideB = TN * kPRowBytes;
  static constexpr int stage = sideA + sideB;
  static constexpr int loadsA = sideA / (kPThreads * 16);
  static constexpr int loadsB = sideB / (kPThreads * 16);
  static constexpr int loads = loadsA + loadsB;  // direct loads per thread per stage
  static constexpr int nb = TN / 64;             // 32-column blocks per wave
};

typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x16 __attribute__((ext_vector_type(16)));

struct ProjArgs {
  const char* a;      // [n, d_in] bf16 or int8
  const char* w;      // [d_out, d_in] bf16 or int8
  const float* sa;    // int8 only: [n] scales of the rows of a
  const float* sw;    // int8 only: [d_out] scales of the rows of w
  void* y;            // [n, d_out], fp32 or bf16
  int64_t n;
  int ld;             // bytes per row of a and w
  int d_out;
  int tiles_m, tiles_n;
  int y_bf16;
};

// bf16 x bf16 -> fp32 or int8 x int8 -> int32, 32x32 output blocks; both
// operands take 16 bytes of k per lane with the same k order, so one LDS
// layout serves both
template <bool I8>
struct PMath {
  using acc_t = f32x16;
  static __device__ __forceinline__ acc_t mma(u32x4 a, u32x4 b, acc_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                   0, 0, 0);
  }
};
template <>
struct PMath<true> {
  using acc_t = i32x16;
  static __device__ __forceinline__ acc_t mma(u32x4 a, u32x4 b, acc_t c) {
    return __builtin_amdgcn_mfma_i32_32x32x32_i8(__builtin_bit_cast(i32x4, a), __builtin_bit_cast(i32x4, b), c, 0,
                                                 0, 0);
  }
};

__device__ __forceinline__ int pswz(int row) { return (row >> 2) & 3; }
__device__ __forceinline__ uint32_t p_lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(ISPA_LDS const void*)p;
}
template <int N>
__device__ __forceinline__ void p_vm_wait() {
  static_assert(N >= 0 && N <= 63, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"i"(N) : "memory");
}

// Direct loads of one side of a stage: rows [row0, row0 + NL * 128) x bytes
// [k0, k0 + 64) of a row-major matrix (ld bytes per row), rows >= rows_end
// zero. Load q of wave w covers 16-byte slot (q * 8 + w) * 64 + lane: row =
// slot / 4, stored chunk = slot % 4.
template <int NL>
__device__ __forceinline__ void p_stage_side(const char* src, int64_t ld, int64_t row0, int64_t rows_end, int k0,
                                             char* dst, int wave, int lane) {
  int64_t nrec = rows_end > row0 ? (rows_end - row0 - 1) * ld + kPRowBytes : 0;
  if (nrec > 0x7fffffff) nrec = 0x7fffffff;
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(src + row0 * ld + k0), 0, (int)nrec, 0x00020000);
#pragma unroll
  for (int q = 0; q < NL; ++q) {
    const int slot = (q * 8 + wave) * 64 + lane;
    const int row = slot >> 2;
    const int c = (slot & 3) ^ pswz(row);
    const int voff = (int)(row * ld + c * 16);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (ISPA_LDS void*)(dst + (q * 8 + wave) * 1024), 16, voff, 0, 0, 0);
  }
}

// Operand read addresses of this lane for stage buffer 0: [block][k-slice].
template <int TN, int MB>
struct PAddr {
  uint32_t a[MB][2];
  uint32_t b[PCfg<TN, MB>::nb][2];
};
template <int TN, int MB>
__device__ __forceinline__ void p_addr(PAddr<TN, MB>& ad, uint32_t base, int wr, int wc, int lane) {
  const int r = lane & 31, h = lane >> 5;
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) {
#pragma unroll
    for (int i = 0; i < MB; ++i) {
      const int row = 32 * MB * wr + 32 * i + r;
      ad.a[i][ks] = base + row * kPRowBytes + (((2 * ks + h) ^ pswz(row)) << 4);
    }
#pragma unroll
    for (int j = 0; j < PCfg<TN, MB>::nb; ++j) {
      const int row = (TN / 2) * wc + 32 * j + r;
      ad.b[j][ks] = base + PCfg<TN, MB>::sideA + row * kPRowBytes + (((2 * ks + h) ^ pswz(row)) << 4);
    }
  }
}

// The operand reads of one 32-byte k slice (inline asm: through the builtin the
// compiler would also wait for the direct loads filling other buffers).
template <int TN, int MB, int IMM>
__device__ __forceinline__ void p_issue(const PAddr<TN, MB>& ad, int ks, u32x4 (&ra)[MB],
                                        u32x4 (&rb)[PCfg<TN, MB>::nb]) {
#pragma unroll
  for (int i = 0; i < MB; ++i)
    asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(ra[i]) : "v"(ad.a[i][ks]), "i"(IMM));
#pragma unroll
  for (int j = 0; j < PCfg<TN, MB>::nb; ++j)
    asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(rb[j]) : "v"(ad.b[j][ks]), "i"(IMM));
}
// Wait for every LDS read of this wave; each operand register is then tied to
// the wait (an empty asm after it, in order), so no use moves above it.
template <int MB, int NB>
__device__ __forceinline__ void p_wait0(u32x4 (&ra)[MB], u32x4 (&rb)[NB]) {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
  for (int i = 0; i < MB; ++i) asm volatile("" : "+v"(ra[i]));
#pragma unroll
  for (int j = 0; j < NB; ++j) asm volatile("" : "+v"(rb[j]));
}

template <int TN, int MB>
struct PTile {
  int64_t row0;  // rows of A / Y
  int col0;      // rows of W / columns of Y
  int steps, wave, lane;
};

template <int TN, int MB>
__device__ __forceinline__ void p_load(const ProjArgs& a, const PTile<TN, MB>& t, char* smem, int s) {
  using C = PCfg<TN, MB>;
  char* d = smem + (s % kPRing) * C::stage;
  p_stage_side<C::loadsA>(a.a, a.ld, t.row0, a.n, s * kPRowBytes, d, t.wave, t.lane);
  p_stage_side<C::loadsB>(a.w, a.ld, t.col0, a.d_out, s * kPRowBytes, d + C::sideA, t.wave, t.lane);
}

// Stage s from ring buffer BUF: loads of stage s + 3, the 2 x nb x 2 MFMAs of
// this wave, then wait for stage s + 1 and synchronise. Buffers 2 and 3 use
// the second address set (LDS offsets are 16-bit immediates).
template <int TN, int MB, bool I8, int BUF>
__device__ __forceinline__ void p_stage(const ProjArgs& a, const PTile<TN, MB>& t, char* smem,
                                        const PAddr<TN, MB>& ad,
                                        typename PMath<I8>::acc_t (&acc)[MB][PCfg<TN, MB>::nb], int s) {
  using C = PCfg<TN, MB>;
  constexpr int kOff = (BUF & 1) * C::stage;
  if (s + 3 < t.steps) p_load<TN, MB>(a, t, smem, s + 3);
  u32x4 ra[MB], rb[C::nb], fa[MB], fb[C::nb];
  p_issue<TN, MB, kOff>(ad, 0, ra, rb);
  p_wait0<MB, C::nb>(ra, rb);
#pragma unroll
  for (int i = 0; i < MB; ++i) fa[i] = ra[i];
#pragma unroll
  for (int j = 0; j < C::nb; ++j) fb[j] = rb[j];
  p_issue<TN, MB, kOff>(ad, 1, ra, rb);
#pragma unroll
  for (int i = 0; i < MB; ++i)
#pragma unroll
    for (int j = 0; j < C::nb; ++j) acc[i][j] = PMath<I8>::mma(fa[i], fb[j], acc[i][j]);
  p_wait0<MB, C::nb>(ra, rb);
#pragma unroll
  for (int i = 0; i < MB; ++i)
#pragma unroll
    for (int j = 0; j < C::nb; ++j) acc[i][j] = PMath<I8>::mma(ra[i], rb[j], acc[i][j]);
  // stage s + 1 must have landed; stages s + 2 and s + 3 may still be in flight
  const int younger = t.steps - (s + 2);
  if (younger >= 2) {
    p_vm_wait<2 * C::loads>();
  } else if (younger == 1) {
    p_vm_wait<C::loads>();
  } else {
    p_vm_wait<0>();
  }
  __builtin_amdgcn_s_barrier();
}

template <int TN, int MB, bool I8>
__global__ __launch_bounds__(kPThreads) __attribute__((amdgpu_waves_per_eu(2))) void proj_kernel(ProjArgs a) {
  using C = PCfg<TN, MB>;
  __shared__ __attribute__((aligned(1024))) char smem[kPRing * C::stage];
  // XCD-aware order: each XCD takes a contiguous run of tiles (row panels of A
  // shared through its L2)
  const int n_items = a.tiles_m * a.tiles_n;
  const int per_xcd = (n_items + 7) / 8;
  const int item = (int)(blockIdx.x % 8) * per_xcd + (int)(blockIdx.x / 8);
  if (item >= n_items) return;
  PTile<TN, MB> t;
  t.row0 = (int64_t)(item / a.tiles_n) * C::tm;
  t.col0 = (item % a.tiles_n) * TN;
  t.lane = threadIdx.x & 63;
  t.wave = threadIdx.x >> 6;
  t.steps = a.ld / kPRowBytes;
  const int wr = t.wave >> 1, wc = t.wave & 1;
  const uint32_t lds0 = p_lds_addr(smem);
  PAddr<TN, MB> ad, ad2;
  p_addr<TN, MB>(ad, lds0, wr, wc, t.lane);
  p_addr<TN, MB>(ad2, lds0 + 2 * C::stage, wr, wc, t.lane);

  typename PMath<I8>::acc_t acc[MB][C::nb];
#pragma unroll
  for (int i = 0; i < MB; ++i)
#pragma unroll
    for (int j = 0; j < C::nb; ++j) acc[i][j] = typename PMath<I8>::acc_t{};

  for (int s = 0; s < 3 && s < t.steps; ++s) p_load<TN, MB>(a, t, smem, s);
  if (t.steps >= 3) {
    p_vm_wait<2 * C::loads>();
  } else if (t.steps == 2) {
    p_vm_wait<C::loads>();
  } else {
    p_vm_wait<0>();
  }
  __builtin_amdgcn_s_barrier();  // stage 0 has landed (vmcnt above)
  for (int s = 0; s < t.steps; s += kPRing) {
    p_stage<TN, MB, I8, 0>(a, t, smem, ad, acc, s);
    if (s + 1 < t.steps) p_stage<TN, MB, I8, 1>(a, t, smem, ad, acc, s + 1);
    if (s + 2 < t.steps) p_stage<TN, MB, I8, 2>(a, t, smem, ad2, acc, s + 2);
    if (s + 3 < t.steps) p_stage<TN, MB, I8, 3>(a, t, smem, ad2, acc, s + 3);
  }

  // lane holds column (lane % 32) and rows 8 (r / 4) + 4 (lane / 32) + r % 4 of each block
#pragma unroll
  for (int j = 0; j < C::nb; ++j) {
    const int ocol = t.col0 + (TN / 2) * wc + 32 * j + (t.lane & 31);
    if (ocol >= a.d_out) continue;
    const float scol = I8 ? a.sw[ocol] : 1.0f;
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t orow = t.row0 + 32 * MB * wr + 32 * i + 8 * (r >> 2) + 4 * (t.lane >> 5) + (r & 3);
        if (orow < a.n) {
          float v;
          if constexpr (I8)
            v = ((float)acc[i][j][r] * a.sa[orow]) * scol;
          else
            v = acc[i][j][r];
          if (a.y_bf16)
            ((__bf16*)a.y)[orow * a.d_out + ocol] = (__bf16)v;
          else
            ((float*)a.y)[orow * a.d_out + ocol] = v;
        }
      }
  }
}

// Codes and scale of one row per wave: pass 1 takes the absmax, pass 2
// re-reads the row (from cache) and writes the codes, 8 values per lane per
// iteration (cols a multiple of 8, rows 16-byte aligned).
template <typename T>
__global__ __launch_bounds__(256) void quant_rows_kernel(const T* __restrict__ x, int64_t rows, int cols,
                                                         int8_t* __restrict__ q, float* __restrict__ scale) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const T* xr = x + row * cols;
  auto load8 = [&](int c, float (&v)[8]) {
    if constexpr (sizeof(T) == 2) {
      const u32x4 u = *(const u32x4*)(xr + c);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[2 * e] = __uint_as_float(u[e] << 16);
        v[2 * e + 1] = __uint_as_float(u[e] & 0xffff0000u);
      }
    } else {
      const f32x4 u0 = *(const f32x4*)(xr + c), u1 = *(const f32x4*)(xr + c + 4);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[e] = u0[e];
        v[4 + e] = u1[e];
      }
    }
  };
  float m = 0.0f;
  for (int c = lane * 8; c < cols; c += 512) {
    float v[8];
    load8(c, v);
#pragma unroll
    for (int e = 0; e < 8; ++e) m = fmaxf(m, fabsf(v[e]));
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
  const float s = m > 0.0f ? m / 127.0f : 1.0f;
  if (lane == 0) scale[row] = s;
  int8_t* qr = q + row * cols;
  for (int c = lane * 8; c < cols; c += 512) {
    float v[8];
    load8(c, v);
    u32x2 out;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      uint32_t word = 0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float r = fminf(fmaxf(rintf(v[4 * h + e] / s), -127.0f), 127.0f);
        word |= ((uint32_t)(int)r & 0xffu) << (8 * e);
      }
      out[h] = word;
    }
    *(u32x2*)(qr + c) = out;
  }
}

}  // namespace

template <int TN, int MB, bool I8>
static void launch_proj_cfg(const ProjArgs& p, hipStream_t stream) {
  const int grid = (p.tiles_m * p.tiles_n + 7) / 8 * 8;
  hipLaunchKernelGGL((proj_kernel<TN, MB, I8>), dim3(grid), dim3(kPThreads), 0, stream, p);
}

static int64_t proj_items(int64_t n, int d_out, int tm, int tn) {
  return ((n + tm - 1) / tm) * ((d_out + tn - 1) / tn);
}

static hipError_t launch_proj(ProjArgs p, bool i8, int d_out, int n_cu, hipStream_t stream) {
  // 256-row tiles of 256 or 128 columns, whichever leaves fewer idle
  // workgroup slots in the last round (ties to the wider tile); the int8 form
  // takes 128 x 128 tiles when 256 x 128 ones would not fill one round, where
  // two workgroups per CU hide its shorter stages better (measured at 4680 x
  // 1536 x 1536: 0.026 ms against 0.030 ms; the bf16 form is slower there)
  const int cu = n_cu > 0 ? n_cu : 256;
  auto fill = [&](int64_t items) { return (double)items / (double)(cu * ((items + cu - 1) / cu)); };
  const int64_t wide = proj_items(p.n, d_out, 256, 256), narrow = proj_items(p.n, d_out, 256, 128);
  int tm = 256, tn = fill(wide) >= fill(narrow) ? 256 : 128;
  if (i8 && narrow < cu) tm = tn = 128;
  p.tiles_m = (int)((p.n + tm - 1) / tm);
  p.tiles_n = (d_out + tn - 1) / tn;
  if (tm == 128)
    launch_proj_cfg<128, 1, true>(p, stream);
  else if (tn == 256)
    i8 ? launch_proj_cfg<256, 2, true>(p, stream) : launch_proj_cfg<256, 2, false>(p, stream);
  else
    i8 ? launch_proj_cfg<128, 2, true>(p, stream) : launch_proj_cfg<128, 2, false>(p, stream);
  return hipGetLastError();
}

hipError_t launch_project(const void* a, const void* w, int64_t n, int d_in, int d_out, void* y, int y_bf16,
                          int n_cu, hipStream_t stream) {
  if (proj_fast_eligible(n, d_in, d_out, false))
    return launch_proj_fast(a, w, nullptr, nullptr, n, d_in, d_out, y, y_bf16, false, n_cu, stream);
  ProjArgs p{};
  p.a = (const char*)a;
  p.w = (const char*)w;
  p.y = y;
  p.n = n;
  p.ld = d_in * 2;
  p.d_out = d_out;
  p.y_bf16 = y_bf16;
  return launch_proj(p, false, d_out, n_cu, stream);
}

hipError_t launch_project_w8a8(const int8_t* qa, const float* sa, const int8_t* qw, const float* sw, int64_t n,
                               int d_in, int d_out, void* y, int y_bf16, int n_cu, hipStream_t stream) {
  if (proj_fast_eligible(n, d_in, d_out, true))
    return launch_proj_fast(qa, qw, sa, sw, n, d_in, d_out, y, y_bf16, true, n_cu, stream);
  ProjArgs p{};
  p.a = (const char*)qa;
  p.w = (const char*)qw;
  p.sa = sa;
  p.sw = sw;
  p.y = y;
  p.n = n;
  p.ld = d_in;
  p.d_out = d_out;
  p.y_bf16 = y_bf16;
  return launch_proj(p, true, d_out, n_cu, stream);
}

hipError_t launch_quantize_rows(const void* x, int x_bf16, int64_t rows, int cols, int8_t* q, float* scale,
                                hipStream_t stream) {
  const unsigned grid = (unsigned)((rows + 3) / 4);
  if (x_bf16)
    hipLaunchKernelGGL(quant_rows_kernel<uint16_t>, dim3(grid), dim3(256), 0, stream, (const uint16_t*)x, rows, cols,
                       q, scale);
  else
    hipLaunchKernelGGL(quant_rows_kernel<float>, dim3(grid), dim3(256), 0, stream, (const float*)x, rows, cols, q,
                       scale);
  return hipGetLastError();
}

}  // namespace ispa
