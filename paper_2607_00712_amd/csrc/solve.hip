// Closed-form modulation dW = (G + lambda I)^-1 C for gfx950 (CDNA4).
//
// Operation (arXiv 2607.00712, Sec. 3.2, Eq. 5): one D x D SPD system with
// D_out right-hand sides, solved once at the end of warmup. The "inversion" is
// a Cholesky factorisation A = L L^T of A = G + lambda I followed by two
// triangular solves L Z = C and L^T dW = Z, all in fp32. Eq. 6's feasibility
// score follows from the same quantities: eps = s - <dW, C> - lambda ||dW||^2.
//
// Blocking: 64 x 64 blocks, nb = D / 64 block rows (ragged last block).
//
// Cholesky, one launch per panel (right-looking, the next panel fused in):
//   launch k (k = -1 .. nb-2) owns the trailing lower block triangle from
//   block k+1 on. Workgroups on the next panel column (r, k+1) apply the rank-64
//   update of panel k to the diagonal block A_{k+1,k+1} (each its own copy in
//   LDS), factor it, invert the factor, and turn their block into
//   L_{r,k+1} = (A_{r,k+1} - L_{r,k} L_{k+1,k}^T) L_{k+1,k+1}^-T. All other
//   workgroups apply A_rt -= L_rk L_tk^T. The diagonal blocks themselves are
//   never overwritten (other workgroups of the same launch read them); their
//   inverses go to Dinv.
// Factor + inverse of one 64 x 64 block (one wave, the others wait): 32 x 32
//   sub-blocks, each factored right-looking with a row per lane in registers
//   and the column multipliers broadcast through LDS, then inverted
//   column-wise; the off-diagonal pieces are 32 x 32 x 32 MFMA products.
// Triangular solves, one launch per block row (right-looking, fused):
//   forward  B_r -= L_{r,i} Z_i for r > i;  tile r = i+1 then forms
//            Z_{i+1} = L_{i+1,i+1}^-1 B_{i+1}
//   backward B_r -= L_{i,r}^T dW_i for r < i; tile r = i-1 then forms
//            dW_{i-1} = L_{i-1,i-1}^-T B_{i-1}
// Every GEMM is fp32 MFMA 32x32x2 (v_mfma_f32_32x32x2f32) on 64 x 64 LDS tiles,
// one 32 x 32 quadrant per wave.
#include "ispa_internal.h"

#include <math.h>

namespace ispa {
namespace {

constexpr int kNb = 64;
constexpr int kThreads = 256;
constexpr int kLd = 65;  // LDS row stride (floats) of a 64 x 64 tile

typedef float Tile[kNb][kLd];

__device__ __forceinline__ f32x16 mfma_f32(float a, float b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}

// acc(32x32) += op(A)[a0 + i, k] . op(B)[k, b0 + j] over k = 0..K-1 for one wave.
// Non-transposed: A_op(i, k) = A[a0 + i][ak + k], B_op(k, j) = B[bk + k][b0 + j].
// TA: A_op(i, k) = A[ak + k][a0 + i].  TB: B_op(k, j) = B[b0 + j][bk + k].
template <bool TA, bool TB>
__device__ __forceinline__ void mma(f32x16& acc, const float (*A)[kLd], int a0, int ak, const float (*B)[kLd],
                                    int b0, int bk, int K, int lane) {
  const int i = lane & 31, kh = lane >> 5;
  for (int k = 0; k < K; k += 2) {
    const float a = TA ? A[ak + k + kh][a0 + i] : A[a0 + i][ak + k + kh];
    const float b = TB ? B[b0 + i][bk + k + kh] : B[bk + k + kh][b0 + i];
    acc = mfma_f32(a, b, acc);
  }
}

// accumulator element r of lane l sits at (row, col) of the 32 x 32 quadrant
__device__ __forceinline__ int acc_row(int r, int lane) { return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3); }

// A 64 x 64 block of a row-major matrix (ld) in flight: four 16-byte pieces per
// thread. Rows >= rows_ok or cols >= cols_ok read as zero (ragged last block).
// Row starts are 16-byte aligned and cols_ok is a multiple of 4 (dimensions are
// multiples of 8). fetch() issues the global loads, put() writes LDS, so the
// loads of several tiles can be in flight together.
struct Frag {
  f32x4 v[4];
};
__device__ __forceinline__ void fetch(Frag& f, const float* src, int64_t ld, int rows_ok, int cols_ok) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int e = threadIdx.x + q * kThreads;
    const int r = e >> 4, c = (e & 15) * 4;
    f.v[q] = (r < rows_ok && c < cols_ok) ? *(const f32x4*)(src + (int64_t)r * ld + c) : f32x4{0.f, 0.f, 0.f, 0.f};
  }
}
__device__ __forceinline__ void put(Tile& t, const Frag& f) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int e = threadIdx.x + q * kThreads;
    const int r = e >> 4, c = (e & 15) * 4;
    t[r][c + 0] = f.v[q][0];
    t[r][c + 1] = f.v[q][1];
    t[r][c + 2] = f.v[q][2];
    t[r][c + 3] = f.v[q][3];
  }
}
__device__ __forceinline__ void load_tile(Tile& t, const float* src, int64_t ld, int rows_ok, int cols_ok) {
  Frag f;
  fetch(f, src, ld, rows_ok, cols_ok);
  put(t, f);
}
__device__ __forceinline__ void store_tile(const Tile& t, float* dst, int64_t ld, int rows_ok, int cols_ok) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int e = threadIdx.x + q * kThreads;
    const int r = e >> 4, c = (e & 15) * 4;
    if (r < rows_ok && c < cols_ok) {
      *(f32x4*)(dst + (int64_t)r * ld + c) = f32x4{t[r][c], t[r][c + 1], t[r][c + 2], t[r][c + 3]};
    }
  }
}

__device__ __forceinline__ float readlane_f(float v, int l) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), l));
}

// Orders the LDS accesses of one wave around this point. A wave's LDS
// operations are performed in issue order, so only the compiler has to be kept
// from moving them.
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

// Scratch of one 32 x 32 factorisation: the current column's multipliers,
// aligned for 16-byte broadcast reads, and a dense copy of the factor.
struct F32Scratch {
  float col[32];
  float Ld[32][32];
};

// One wave: factor the 32 x 32 block S[o..o+31][o..o+31] (lower part) in place
// (zero above) and write its inverse, lower triangular, to M[o..][o..].
// Right-looking, a row per lane (lanes 32..63 mirror 0..31): at step j lane i
// keeps a[m] = A[i][j + m] in registers; the multipliers l_cj of column j are
// broadcast through LDS (lane c writes its l_cj at col[c - j - 1], everybody
// reads col[0..31] with 16-byte loads) and the update shifts the row by one, so
// register indices stay static inside a compact loop. Pivots use the hardware
// square root and reciprocal (about 1 ulp). The inverse is formed column-wise
// (a column per lane) from the dense copy of the factor. Sets *bad on a
// non-positive pivot.
__device__ void factor32(Tile& S, Tile& M, int o, int lane, int* bad, F32Scratch& w) {
  const int i = lane & 31;
  const bool lo = lane < 32;
  float a[32];
#pragma unroll
  for (int c = 0; c < 32; ++c) a[c] = S[o + i][o + c];
  int neg = 0;
  for (int j = 0; j < 32; ++j) {
    float piv = readlane_f(a[0], j);
    neg |= !(piv > 0.f);
    piv = piv > 0.f ? piv : 1.f;
    const float ljj = __builtin_amdgcn_sqrtf(piv);
    const float lij = i > j ? a[0] * __builtin_amdgcn_rcpf(ljj) : (i == j ? ljj : 0.f);
    if (lo) {
      w.Ld[i][j] = lij;
      if (i > j) w.col[i - j - 1] = lij;
    }
    wave_sync();
    float cb[32];
#pragma unroll
    for (int m = 0; m < 32; m += 4) {
      const f32x4 v = *(const f32x4*)(&w.col[m]);
      cb[m] = v[0];
      cb[m + 1] = v[1];
      cb[m + 2] = v[2];
      cb[m + 3] = v[3];
    }
    // a[m] <- A[i][j + 1 + m] - l_ij l_{j+1+m, j}; entries past column 31 are
    // stale but never reach a[0]
#pragma unroll
    for (int m = 0; m < 31; ++m) a[m] = fmaf(-lij, cb[m], a[m + 1]);
    a[31] = 0.f;
    wave_sync();
  }
  if (neg && lane == 0) *bad = 1;
  // factor back into S (zero above the diagonal)
  if (lo) {
#pragma unroll
    for (int c = 0; c < 32; ++c) S[o + i][o + c] = w.Ld[i][c];
  }
  wave_sync();
  // inverse: lane j owns column j; M[r][j] = (d_rj - sum_{p<r} L_rp M_pj) / L_rr
  const int j = i;
  float m[32];
#pragma unroll
  for (int r = 0; r < 32; ++r) {
    float acc = r == j ? 1.f : 0.f;
#pragma unroll
    for (int p = 0; p < r; ++p) acc = fmaf(-w.Ld[r][p], m[p], acc);
    m[r] = acc * __builtin_amdgcn_rcpf(w.Ld[r][r]);
  }
  if (lo) {
#pragma unroll
    for (int r = 0; r < 32; ++r) M[o + r][o + j] = m[r];
  }
  wave_sync();
}

// Factor the 64 x 64 SPD block in S (lower part valid) into L (in place, zero
// above) and write L^-1 to M. All threads call; wave 0 works.
__device__ void factor64(Tile& S, Tile& M, Tile& T, int nb, int* bad, F32Scratch& w) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  // a ragged last block: identity beyond nb keeps the factorisation defined
  for (int e = threadIdx.x; e < kNb * kNb; e += kThreads) {
    const int r = e >> 6, c = e & 63;
    if (r >= nb || c >= nb) S[r][c] = r == c ? 1.f : 0.f;
    M[r][c] = 0.f;
  }
  __syncthreads();
  if (wave == 0) {
    factor32(S, M, 0, lane, bad, w);
    // L10 = S10 . M00^T
    f32x16 acc = {};
    mma<false, true>(acc, S, 32, 0, M, 0, 0, 32, lane);
    wave_sync();
#pragma unroll
    for (int r = 0; r < 16; ++r) S[32 + acc_row(r, lane)][lane & 31] = acc[r];
    wave_sync();
    // S11 -= L10 . L10^T
    acc = f32x16{};
    mma<false, true>(acc, S, 32, 0, S, 32, 0, 32, lane);
#pragma unroll
    for (int r = 0; r < 16; ++r) S[32 + acc_row(r, lane)][32 + (lane & 31)] -= acc[r];
    wave_sync();
    factor32(S, M, 32, lane, bad, w);
    // M10 = -M11 . L10 . M00 : T = L10 . M00, then M10 = -M11 . T
    acc = f32x16{};
    mma<false, false>(acc, S, 32, 0, M, 0, 0, 32, lane);
#pragma unroll
    for (int r = 0; r < 16; ++r) T[acc_row(r, lane)][lane & 31] = acc[r];
    wave_sync();
    acc = f32x16{};
    mma<false, false>(acc, M, 32, 32, T, 0, 0, 32, lane);
#pragma unroll
    for (int r = 0; r < 16; ++r) M[32 + acc_row(r, lane)][lane & 31] = -acc[r];
  }
  __syncthreads();
}

// Quadrant product over a full 64-deep tile pair, one quadrant per wave:
// acc = op(A)[wr.., :] op(B)[:, wc..]
template <bool TA, bool TB>
__device__ __forceinline__ f32x16 quad(const Tile& A, const Tile& B) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  f32x16 acc = {};
  mma<TA, TB>(acc, A, (wave >> 1) * 32, 0, B, (wave & 1) * 32, 0, kNb, lane);
  return acc;
}
__device__ __forceinline__ void quad_store(Tile& D, const f32x16& acc, float sign, bool add) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r0 = (wave >> 1) * 32, c0 = (wave & 1) * 32;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    float& d = D[r0 + acc_row(r, lane)][c0 + (lane & 31)];
    d = add ? d + sign * acc[r] : sign * acc[r];
  }
}

__device__ __forceinline__ void tri_index(int t, int& ti, int& tj) {
  ti = (int)((sqrtf(8.f * t + 1.f) - 1.f) * 0.5f);
  while ((ti + 1) * (ti + 2) / 2 <= t) ++ti;
  while (ti * (ti + 1) / 2 > t) --ti;
  tj = t - ti * (ti + 1) / 2;
}

// L = lower(G) + lambda I (upper part zero), Bw = C, status = 0.
__global__ void solve_init_kernel(const float* G, float* L, const float* C, float* Bw, int n, int n_out,
                                  float lambda, int* status) {
  const int64_t nn = (int64_t)n * n, nc = (int64_t)n * n_out;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nn + nc;
       i += (int64_t)gridDim.x * blockDim.x) {
    if (i < nn) {
      const int r = (int)(i / n), c = (int)(i % n);
      L[i] = c < r ? G[i] : (c == r ? G[i] + lambda : 0.f);
    } else {
      Bw[i - nn] = C[i - nn];
    }
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) *status = 0;
}

// Cholesky launch k: trailing lower block triangle from block k+1.
__global__ __launch_bounds__(kThreads) void chol_step_kernel(float* L, float* Dinv, int n, int k, int* status) {
  __shared__ Tile S, M, T, U, V;
  __shared__ __attribute__((aligned(16))) F32Scratch fw;
  __shared__ int bad;
  const int nblk = (n + kNb - 1) / kNb;
  int ti, tj;
  if (k < 0) {
    ti = blockIdx.x;  // first launch: the first panel column only
    tj = 0;
  } else {
    tri_index(blockIdx.x, ti, tj);
  }
  const int r = k + 1 + ti, t = k + 1 + tj;  // block coordinates, r >= t
  if (r >= nblk) return;
  const int rr = min(kNb, n - r * kNb), rt = min(kNb, n - t * kNb);
  float* Lrt = L + (int64_t)r * kNb * n + t * kNb;
  if (threadIdx.x == 0) bad = 0;

  if (t > k + 1) {
    // plain trailing update A_rt -= L_rk L_tk^T
    Frag fu, fv, ft;
    fetch(fu, L + (int64_t)r * kNb * n + k * kNb, n, rr, kNb);
    fetch(fv, L + (int64_t)t * kNb * n + k * kNb, n, rt, kNb);
    fetch(ft, Lrt, n, rr, rt);
    put(U, fu);
    put(V, fv);
    put(T, ft);
    __syncthreads();
    quad_store(T, quad<false, true>(U, V), -1.f, true);
    __syncthreads();
    store_tile(T, Lrt, n, rr, rt);
    return;
  }
  // next panel column: updated diagonal block, factor, inverse
  const int d = k + 1;
  const int nd = min(kNb, n - d * kNb);
  const bool off = r != d;
  Frag fs, fv, ft, fu;
  fetch(fs, L + (int64_t)d * kNb * n + d * kNb, n, nd, nd);
  if (k >= 0) fetch(fv, L + (int64_t)d * kNb * n + k * kNb, n, nd, kNb);
  if (off) {
    fetch(ft, Lrt, n, rr, nd);
    if (k >= 0) fetch(fu, L + (int64_t)r * kNb * n + k * kNb, n, rr, kNb);
  }
  put(S, fs);
  if (k >= 0) put(V, fv);
  __syncthreads();
  if (k >= 0) {
    quad_store(S, quad<false, true>(V, V), -1.f, true);
    __syncthreads();
  }
  factor64(S, M, T, nd, &bad, fw);
  if (!off) {
    store_tile(M, Dinv + (int64_t)d * kNb * kNb, kNb, kNb, kNb);
    if (threadIdx.x == 0 && bad) atomicOr(status, 1);
    return;
  }
  // L_rd = (A_rd - L_rk L_dk^T) . M^T
  put(T, ft);
  if (k >= 0) put(U, fu);
  __syncthreads();
  if (k >= 0) {
    quad_store(T, quad<false, true>(U, V), -1.f, true);
    __syncthreads();
  }
  const f32x16 x = quad<false, true>(T, M);
  __syncthreads();
  quad_store(T, x, 1.f, false);
  __syncthreads();
  store_tile(T, Lrt, n, rr, nd);
}

// Forward solve launch i (i = -1 .. nb-2): B_r -= L_{r,i} Z_i for r > i; tile
// r = i+1 forms Z_{i+1} = Dinv_{i+1} B_{i+1}. Grid: (nb-1-i) x column tiles.
__global__ __launch_bounds__(kThreads) void trsm_fwd_kernel(const float* L, const float* Dinv, float* Bw, float* Z,
                                                           int n, int n_out, int i) {
  __shared__ Tile A, X, Bt;
  const int nblk = (n + kNb - 1) / kNb;
  const int ctiles = (n_out + kNb - 1) / kNb;
  const int r = i + 1 + blockIdx.x / ctiles;
  const int c = blockIdx.x % ctiles;
  if (r >= nblk) return;
  const int rr = min(kNb, n - r * kNb), cc = min(kNb, n_out - c * kNb);
  float* Br = Bw + (int64_t)r * kNb * n_out + c * kNb;
  const bool last = r == i + 1;
  Frag fb, fa, fx, fd;
  fetch(fb, Br, n_out, rr, cc);
  if (i >= 0) {
    const int ri = min(kNb, n - i * kNb);
    fetch(fa, L + (int64_t)r * kNb * n + i * kNb, n, rr, ri);
    fetch(fx, Z + (int64_t)i * kNb * n_out + c * kNb, n_out, ri, cc);
  }
  if (last) fetch(fd, Dinv + (int64_t)r * kNb * kNb, kNb, kNb, kNb);
  put(Bt, fb);
  if (i >= 0) {
    put(A, fa);
    put(X, fx);
  }
  __syncthreads();
  if (i >= 0) {
    quad_store(Bt, quad<false, false>(A, X), -1.f, true);
    __syncthreads();
  }
  if (last) {
    put(A, fd);
    __syncthreads();
    const f32x16 z = quad<false, false>(A, Bt);
    __syncthreads();
    quad_store(Bt, z, 1.f, false);
    __syncthreads();
    store_tile(Bt, Z + (int64_t)r * kNb * n_out + c * kNb, n_out, rr, cc);
  } else {
    store_tile(Bt, Br, n_out, rr, cc);
  }
}

// Backward solve launch i (i = nb .. 1), in place on W (holds Z, becomes dW):
// W_r -= L_{i,r}^T W_i for r < i; tile r = i-1 forms W_{i-1} = Dinv_{i-1}^T W_{i-1}.
__global__ __launch_bounds__(kThreads) void trsm_bwd_kernel(const float* L, const float* Dinv, float* W, int n,
                                                           int n_out, int i) {
  __shared__ Tile A, X, Bt;
  const int nblk = (n + kNb - 1) / kNb;
  const int ctiles = (n_out + kNb - 1) / kNb;
  const int r = i - 1 - blockIdx.x / ctiles;
  const int c = blockIdx.x % ctiles;
  if (r < 0) return;
  const int rr = min(kNb, n - r * kNb), cc = min(kNb, n_out - c * kNb);
  float* Wr = W + (int64_t)r * kNb * n_out + c * kNb;
  const bool last = r == i - 1;
  Frag fb, fa, fx, fd;
  fetch(fb, Wr, n_out, rr, cc);
  if (i < nblk) {
    const int ri = min(kNb, n - i * kNb);
    fetch(fa, L + (int64_t)i * kNb * n + r * kNb, n, ri, rr);  // L_{i,r}, used transposed
    fetch(fx, W + (int64_t)i * kNb * n_out + c * kNb, n_out, ri, cc);
  }
  if (last) fetch(fd, Dinv + (int64_t)r * kNb * kNb, kNb, kNb, kNb);
  put(Bt, fb);
  if (i < nblk) {
    put(A, fa);
    put(X, fx);
  }
  __syncthreads();
  if (i < nblk) {
    quad_store(Bt, quad<true, false>(A, X), -1.f, true);
    __syncthreads();
  }
  if (last) {
    put(A, fd);
    __syncthreads();
    const f32x16 z = quad<true, false>(A, Bt);
    __syncthreads();
    quad_store(Bt, z, 1.f, false);
    __syncthreads();
  }
  store_tile(Bt, Wr, n_out, rr, cc);
}

// scalars[0] = <dW, C>, scalars[1] = ||dW||^2 (zeroed by the first block, then
// accumulated; launched as a single pass after zeroing)
__global__ __launch_bounds__(kThreads) void eps_kernel(const float* dw, const float* C, int64_t n, double* scalars) {
  __shared__ double red[2][kThreads / 64];
  double a = 0, b = 0;
  for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n; i += (int64_t)gridDim.x * kThreads) {
    const double w = dw[i];
    a += w * (double)C[i];
    b += w * w;
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    a += __shfl_xor(a, o);
    b += __shfl_xor(b, o);
  }
  if ((threadIdx.x & 63) == 0) {
    red[0][threadIdx.x >> 6] = a;
    red[1][threadIdx.x >> 6] = b;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    double ta = 0, tb = 0;
    for (int w = 0; w < kThreads / 64; ++w) {
      ta += red[0][w];
      tb += red[1][w];
    }
    atomicAdd(&scalars[0], ta);
    atomicAdd(&scalars[1], tb);
  }
}

__global__ void zero_scalars_kernel(double* s) {
  if (threadIdx.x < 2) s[threadIdx.x] = 0.0;
}

}  // namespace

size_t solve_dinv_bytes(int d) {
  const int nblk = (d + kNb - 1) / kNb;
  return (size_t)nblk * kNb * kNb * sizeof(float);
}

hipError_t launch_solve(const float* G, const float* C, int d, int d_out, float lambda, float* delta_w,
                        const SolveWork& w, hipStream_t stream) {
  const int nblk = (d + kNb - 1) / kNb;
  const int ctiles = (d_out + kNb - 1) / kNb;
  {
    const int64_t total = (int64_t)d * d + (int64_t)d * d_out;
    int grid = (int)((total + 255) / 256);
    if (grid > 8192) grid = 8192;
    hipLaunchKernelGGL(solve_init_kernel, dim3(grid), dim3(256), 0, stream, G, w.L, C, w.work, d, d_out, lambda,
                       w.status);
  }
  for (int k = -1; k <= nblk - 2; ++k) {
    const int m = nblk - 1 - k;  // blocks in the trailing triangle
    const int grid = k < 0 ? nblk : m * (m + 1) / 2;
    hipLaunchKernelGGL(chol_step_kernel, dim3(grid), dim3(kThreads), 0, stream, w.L, w.dinv, d, k, w.status);
  }
  for (int i = -1; i <= nblk - 2; ++i) {
    const int rows = i < 0 ? 1 : nblk - 1 - i;
    hipLaunchKernelGGL(trsm_fwd_kernel, dim3(rows * ctiles), dim3(kThreads), 0, stream, w.L, w.dinv, w.work,
                       delta_w, d, d_out, i);
  }
  for (int i = nblk; i >= 1; --i) {
    const int rows = i == nblk ? 1 : i;
    hipLaunchKernelGGL(trsm_bwd_kernel, dim3(rows * ctiles), dim3(kThreads), 0, stream, w.L, w.dinv, delta_w, d,
                       d_out, i);
  }
  hipLaunchKernelGGL(zero_scalars_kernel, dim3(1), dim3(64), 0, stream, w.scalars);
  const int64_t n = (int64_t)d * d_out;
  int eg = (int)((n + kThreads - 1) / kThreads);
  if (eg > 256) eg = 256;  // one fp64 atomic pair per block
  hipLaunchKernelGGL(eps_kernel, dim3(eg), dim3(kThreads), 0, stream, delta_w, C, n, w.scalars);
  return hipGetLastError();
}

}  // namespace ispa
