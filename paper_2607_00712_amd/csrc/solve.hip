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
//   sub-blocks, each reduced in registers with the pivot row broadcast by
//   readlane, the inverse formed in the same instructions by the other half of
//   the wave; the off-diagonal pieces are 32 x 32 x 32 MFMA products.
// Triangular solves in block LDL^T form over 256-blocks (details below): the
//   inverses X_I of the 256 x 256 diagonal blocks of L and P_I = X_I^T X_I,
//   Lh = L diag(X_I) below the 256-block diagonal (its transpose mirrored into
//   the upper part), then one right-looking rank-256 GEMM launch per block for
//   the forward and for the backward sweep, with no diagonal work in them.
// Every product is fp32 MFMA (v_mfma_f32_32x32x2f32); the sweeps' GEMM stages
// its operands HBM -> LDS with direct buffer loads in a 4-deep ring.
// Several layers at once (the end of warmup solves every layer): every kernel
// takes its layer from the last grid dimension and offsets its workspace
// pointers by the layers' workspace stride (dW by its own stride), so one
// launch per step covers all layers with each layer's arithmetic unchanged.
#include "ispa_internal.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <mutex>
#include <utility>

namespace ispa {
namespace {

constexpr int kNb = 64;
constexpr int kSup = 4;  // panels per super-panel of the deferred trailing update
constexpr int kThreads = 256;
constexpr int kLd = 65;  // LDS row stride (floats) of a 64 x 64 tile

typedef float Tile[kNb][kLd];

// Batched solves (one per layer, the layer from the last grid dimension): the
// layers' workspaces are `bytes` apart.
template <class T>
__device__ __forceinline__ T* at_layer(T* p, int64_t bytes, int layer) {
  return (T*)((char*)p + bytes * layer);
}

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

// 16 x 16 pieces (v_mfma_f32_16x16x4f32): lane l supplies A[l % 16][k + l / 16]
// and B[k + l / 16][l % 16]; accumulator element r of lane l sits at row
// 4 (l / 16) + r, column l % 16.
// acc = op(A)[a0 .., ak ..] op(B)[bk .., b0 ..] over K, same conventions as mma.
template <bool TA, bool TB, int K>
__device__ __forceinline__ f32x4 mma16(const float (*A)[kLd], int a0, int ak, const float (*B)[kLd], int b0, int bk,
                                       int lane) {
  const int i = lane & 15, kq = lane >> 4;
  f32x4 acc = {};
#pragma unroll
  for (int k = 0; k < K; k += 4) {
    const float a = TA ? A[ak + k + kq][a0 + i] : A[a0 + i][ak + k + kq];
    const float b = TB ? B[b0 + i][bk + k + kq] : B[bk + k + kq][b0 + i];
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc, 0, 0, 0);
  }
  return acc;
}
// D[r0 ..][c0 ..] (16 x 16) = sign * acc, or += sign * acc
__device__ __forceinline__ void put16(Tile& D, int r0, int c0, const f32x4& acc, float sign, bool add, int lane) {
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    float& d = D[r0 + 4 * (lane >> 4) + r][c0 + (lane & 15)];
    d = add ? d + sign * acc[r] : sign * acc[r];
  }
}

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

// One wave: factor the N x N SPD block S[o..o+N-1][o..o+N-1] (N = 16 or 32,
// lower part valid) into L, in place with zeros above the diagonal, and write
// L^-1 (lower triangular) to M[o..][o..]. No LDS traffic inside the elimination:
//   lanes 0..N-1    x = row i of the symmetric matrix being reduced,
//   lanes N..2N-1   x = column i - N of the inverse being formed by forward
//                   substitution, starting from the unit vector
// (for N = 16 lanes 32..63 repeat lanes 0..31 and store nothing).
// At step j the pivot p_j = (row j)[j] and s_c = (row j)[c] = (column j)[c]
// (symmetry) come from lane j by readlane, and both kinds of lane apply the
// same update x[c] -= (x[j] / p_j) s_c for c > j: the Schur complement for a
// row, the substitution step m_c -= L_cj m_j / L_jj for an inverse column.
// Afterwards L[i][j] = x[j] / sqrt(p_j) (j < i), L[i][i] = sqrt(p_i) and
// L^-1[r][col] = x[r] / sqrt(p_r). Hardware square root and reciprocal (about
// 1 ulp). Sets *bad on a non-positive pivot (then replaced by 1).
template <int N>
__device__ __forceinline__ void factor_reg(Tile& S, Tile& M, int o, int lane, int* bad) {
  const int i = lane % N;
  const bool lo = (lane / N) % 2 == 0;
  float x[N];
#pragma unroll
  for (int c = 0; c < N; ++c) {
    float v = S[o + max(i, c)][o + min(i, c)];
    asm volatile("" : "+v"(v));  // every lane loads: no branch around the read
    x[c] = lo ? v : (c == i ? 1.f : 0.f);
  }
  float lj[N];
  int neg = 0;
#pragma unroll
  for (int j = 0; j < N; ++j) {
    float piv = readlane_f(x[j], j);
    neg |= !(piv > 0.f);
    piv = piv > 0.f ? piv : 1.f;
    lj[j] = piv;
    // the pivot row first (independent readlanes), then the updates
    float sr[N];
#pragma unroll
    for (int c = j + 1; c < N; ++c) sr[c] = readlane_f(x[c], j);
    const float coef = x[j] * __builtin_amdgcn_rcpf(piv);
#pragma unroll
    for (int c = j + 1; c < N; ++c) x[c] = fmaf(-coef, sr[c], x[c]);
  }
  if (neg && lane == 0) *bad = 1;
  // one store per element: row i of L for the row lanes, column i of L^-1 for the rest
  float* dst = lo ? &S[o + i][o] : &M[o][o + i];
  const int step = lo ? 1 : kLd;
  if (lane < 2 * N) {
#pragma unroll
    for (int c = 0; c < N; ++c) {
      const float l = __builtin_amdgcn_sqrtf(lj[c]);
      const float v = x[c] * __builtin_amdgcn_rcpf(l);
      dst[c * step] = lo ? (c < i ? v : (c == i ? l : 0.f)) : (c >= i ? v : 0.f);
    }
  }
  wave_sync();
}

// One wave: the 32 x 32 factor and inverse at offset o from two 16 x 16 register
// factors: L00 and M00; L10 = S10 M00^T; S11 -= L10 L10^T with T = L10 M00
// beside it (T in the upper-right 16 x 16 of this block of M, zero again at the
// end); L11 and M11; M10 = -M11 T. The 16-wide eliminations issue a third of the
// readlanes and FMAs of one 32-wide elimination, and the products are four
// 16x16x4 MFMAs each.
__device__ __forceinline__ void factor32(Tile& S, Tile& M, int o, int lane, int* bad) {
  factor_reg<16>(S, M, o, lane, bad);
  {
    const f32x4 l10 = mma16<false, true, 16>(S, o + 16, o, M, o, o, lane);
    put16(S, o + 16, o, l10, 1.f, false, lane);  // in place: its reads are issued before
  }
  wave_sync();
  {
    const f32x4 u = mma16<false, true, 16>(S, o + 16, o, S, o + 16, o, lane);
    const f32x4 t = mma16<false, false, 16>(S, o + 16, o, M, o, o, lane);
    put16(S, o + 16, o + 16, u, -1.f, true, lane);
    put16(M, o, o + 16, t, 1.f, false, lane);
  }
  wave_sync();
  factor_reg<16>(S, M, o + 16, lane, bad);
  {
    const f32x4 m10 = mma16<false, false, 16>(M, o + 16, o + 16, M, o + 16, o, lane);
    put16(M, o + 16, o, m10, -1.f, false, lane);
    put16(M, o, o + 16, f32x4{}, 1.f, false, lane);
  }
  wave_sync();
}

// Factor the 64 x 64 SPD block in S (lower part valid, zero above) into L (in
// place) and write L^-1 to M; T is scratch. All threads call; wave 0 factors.
// With P given, waves 1..3 meanwhile apply P -= Q R^T (the panel block's own
// rank-64 update, independent of the factor), quadrant q on wave 1 + q % 3.
__device__ void factor64(Tile& S, Tile& M, Tile& T, int nb, int* bad, Tile* P, const Tile* Q, const Tile* R) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  // a ragged last block: identity beyond nb keeps the factorisation defined
  if (nb < kNb) {
    for (int e = threadIdx.x; e < kNb * kNb; e += kThreads) {
      const int r = e >> 6, c = e & 63;
      if (r >= nb || c >= nb) S[r][c] = r == c ? 1.f : 0.f;
    }
  }
  // the quadrant of L^-1 above the diagonal; factor32 writes the other three
  for (int e = threadIdx.x; e < 32 * 32; e += kThreads) M[e >> 5][32 + (e & 31)] = 0.f;
  __syncthreads();
  // the 32 x 32 products below are split over the four waves, 16 x 16 each
  const int qr = 16 * (wave >> 1), qc = 16 * (wave & 1);
  if (wave == 0) {
    factor32(S, M, 0, lane, bad);
  } else if (P) {
    for (int q = wave - 1; q < 4; q += 3) {
      const int r0 = (q >> 1) * 32, c0 = (q & 1) * 32;
      f32x16 acc = {};
      mma<false, true>(acc, *Q, r0, 0, *R, c0, 0, kNb, lane);
#pragma unroll
      for (int r = 0; r < 16; ++r) (*P)[r0 + acc_row(r, lane)][c0 + (lane & 31)] -= acc[r];
    }
  }
  __syncthreads();
  // L10 = S10 . M00^T (in place: all reads before the stores)
  {
    const f32x4 acc = mma16<false, true, 32>(S, 32 + qr, 0, M, qc, 0, lane);
    __syncthreads();
    put16(S, 32 + qr, qc, acc, 1.f, false, lane);
  }
  __syncthreads();
  // S11 -= L10 . L10^T and T = L10 . M00 (for M10 = -M11 . L10 . M00)
  {
    const f32x4 u = mma16<false, true, 32>(S, 32 + qr, 0, S, 32 + qc, 0, lane);
    const f32x4 t = mma16<false, false, 32>(S, 32 + qr, 0, M, qc, 0, lane);
    put16(S, 32 + qr, 32 + qc, u, -1.f, true, lane);
    put16(T, qr, qc, t, 1.f, false, lane);
  }
  __syncthreads();
  if (wave == 0) factor32(S, M, 32, lane, bad);
  __syncthreads();
  // M10 = -M11 . T
  put16(M, 32 + qr, qc, mma16<false, false, 32>(M, 32 + qr, 32, T, qc, 0, lane), -1.f, false, lane);
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

// L = lower(G) + lambda I with zeros above the diagonal up to the end of the
// row's 256-block (the part above the 256-block diagonal is never read before
// the mirror of Lh overwrites it), status = 0. Row blockIdx.x, four columns per
// thread (n is a multiple of 4); only G's lower triangle is read.
__global__ void solve_init_kernel(const float* G, float* L, int n, float lambda, int* status, int64_t ws) {
  G = at_layer(G, ws, blockIdx.y);
  L = at_layer(L, ws, blockIdx.y);
  status = at_layer(status, ws, blockIdx.y);
  constexpr int kBlock = 256;  // the sweeps' block size
  const int r = blockIdx.x;
  const int end = min(n, (r / kBlock + 1) * kBlock);
  const float* g = G + (int64_t)r * n;
  float* l = L + (int64_t)r * n;
  for (int c = threadIdx.x * 4; c < end; c += blockDim.x * 4) {
    f32x4 v = c <= r ? *(const f32x4*)(g + c) : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if (c + j > r) v[j] = 0.f;
      else if (c + j == r) v[j] += lambda;
    }
    *(f32x4*)(l + c) = v;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) *status = 0;
}

// Trailing update by the panels p0 .. p0 + NP - 1 of a 2 x 2 group of 64-blocks
// with top-left block (R, T), R >= T: A_rt -= L_rp L_tp^T for p in order, block
// (R + w / 2, T + w % 2) on wave w (blocks past the matrix, above the diagonal
// or in a column >= t_end are skipped). The four waves share L_rp (rows of
// blocks R, R + 1) and L_tp staged in LDS, one panel at a time, the next
// panel's tiles loaded into registers during this one's MFMAs; each wave's C
// block stays in registers from the first panel to the last. Each panel's
// product is subtracted on its own, in panel order, so the result is bit for
// bit that of one launch per panel.
template <int NP>
__device__ __forceinline__ void trailing_2x2(float* L, int n, int nblk, int p0, int R, int T, int t_end, Tile* tiles) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int l32 = lane & 31, h = lane >> 5;
  float (*Ub)[kLd] = tiles[0];  // [128][kLd]: rows of blocks R, R + 1 (two consecutive tiles)
  float (*Vb)[kLd] = tiles[2];  // [128][kLd]: rows of blocks T, T + 1
  const int br = R + (wave >> 1), bc = T + (wave & 1);
  const bool mine = br < nblk && bc <= br && bc < t_end;
  const int rows_r0 = min(kNb, n - R * kNb), rows_r1 = min(kNb, n - (R + 1) * kNb);
  const int rows_t0 = min(kNb, n - T * kNb), rows_t1 = min(kNb, n - (T + 1) * kNb);
  Frag f0, f1, f2, f3;
  fetch(f0, L + (int64_t)R * kNb * n + p0 * kNb, n, rows_r0, kNb);
  fetch(f1, L + (int64_t)(R + 1) * kNb * n + p0 * kNb, n, rows_r1, kNb);
  fetch(f2, L + (int64_t)T * kNb * n + p0 * kNb, n, rows_t0, kNb);
  fetch(f3, L + (int64_t)(T + 1) * kNb * n + p0 * kNb, n, rows_t1, kNb);
  float c[2][2][16];
  if (mine) {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = br * kNb + 32 * i + acc_row(r, lane), col = bc * kNb + 32 * j + l32;
          c[i][j][r] = row < n && col < n ? L[(int64_t)row * n + col] : 0.f;
        }
  }
  const int qr = (wave >> 1) * kNb, qc = (wave & 1) * kNb;
#pragma unroll
  for (int pi = 0; pi < NP; ++pi) {
    const int p = p0 + pi;
    if (pi > 0) __syncthreads();  // every wave is done with the previous panel's tiles
    put(tiles[0], f0);
    put(tiles[1], f1);
    put(tiles[2], f2);
    put(tiles[3], f3);
    __syncthreads();
    if (pi + 1 < NP) {
      fetch(f0, L + (int64_t)R * kNb * n + (p + 1) * kNb, n, rows_r0, kNb);
      fetch(f1, L + (int64_t)(R + 1) * kNb * n + (p + 1) * kNb, n, rows_r1, kNb);
      fetch(f2, L + (int64_t)T * kNb * n + (p + 1) * kNb, n, rows_t0, kNb);
      fetch(f3, L + (int64_t)(T + 1) * kNb * n + (p + 1) * kNb, n, rows_t1, kNb);
    }
    if (mine) {
      f32x16 acc[2][2] = {};
#pragma unroll
      for (int kk = 0; kk < kNb; kk += 2) {
        float a[2], b[2];
#pragma unroll
        for (int i = 0; i < 2; ++i) a[i] = Ub[qr + 32 * i + l32][kk + h];
#pragma unroll
        for (int j = 0; j < 2; ++j) b[j] = Vb[qc + 32 * j + l32][kk + h];
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j) acc[i][j] = mfma_f32(a[i], b[j], acc[i][j]);
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) c[i][j][r] -= acc[i][j][r];
    }
  }
  if (!mine) return;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = br * kNb + 32 * i + acc_row(r, lane), col = bc * kNb + 32 * j + l32;
        if (row < n && col < n) L[(int64_t)row * n + col] = c[i][j][r];
      }
}

// The deferred update of a super-panel of kSup panels (p0 .. p0 + kSup - 1): the
// trailing triangle from block e on (rows r >= t >= e) in 2 x 2 groups.
__global__ __launch_bounds__(kThreads) void chol_trail_kernel(float* L, int n, int p0, int e, int64_t ws) {
  __shared__ __attribute__((aligned(16))) Tile tiles[4];
  L = at_layer(L, ws, blockIdx.y);
  const int nblk = (n + kNb - 1) / kNb;
  int ti, tj;
  tri_index((int)blockIdx.x, ti, tj);
  trailing_2x2<kSup>(L, n, nblk, p0, e + 2 * ti, e + 2 * tj, nblk, tiles);
}

// Panel-group updates that ride along in a single layer's panel launches (the
// look-ahead form of the factorisation), kLa panels at a time. Band b is block
// columns kLa b + 1 .. kLa b + kLa; task t applies the kLa panels of group
// sp[t] (panels kLa sp[t] ..) to every block of band band[t] at or below the
// diagonal, in groups[t] 2 x 2 groups, group column by group column. The
// tasks' workgroups follow the launch's `trail` groups.
constexpr int kLa = 2;
constexpr int kMaxTasks = 64;
struct CholExtra {
  int trail;  // -1: no tasks
  int n_tasks;
  int band[kMaxTasks], sp[kMaxTasks], groups[kMaxTasks];
};

// What workgroup wg of Cholesky launch k works on; the kernel and the host
// check of the look-ahead schedule share this decode. kind 0: the block of the
// next panel column in row R (column T = k + 1), which receives panel k when
// the launch applies it; kind 1: the 2 x 2 group of blocks with top-left
// (R, T), of which the blocks at or below the diagonal, inside the matrix and
// left of column t_end receive the np panels p0 ..; kind -1: nothing.
struct CholWork {
  int kind, R, T, p0, np, t_end;
};
__host__ __device__ inline CholWork chol_work_of(int wg, int nblk, int k, int t_end, int split, const CholExtra& ex) {
  CholWork w = {-1, 0, 0, 0, 0, 0};
  const int m = split == 2 ? nblk - 2 - k : nblk - 1 - k;  // panel-column workgroups of this launch
  if (ex.trail >= 0 && wg >= m + ex.trail) {
    int idx = wg - m - ex.trail;
    for (int t = 0; t < ex.n_tasks; ++t) {
      if (idx < ex.groups[t]) {
        const int e = ex.band[t] * kLa + 1, end = e + kLa < nblk ? e + kLa : nblk;
        for (int T = e; T < end; T += 2) {
          const int gr = (nblk - T + 1) / 2;  // groups of this group column
          if (idx < gr) {
            w = CholWork{1, T + 2 * idx, T, ex.sp[t] * kLa, kLa, end};
            return w;
          }
          idx -= gr;
        }
        return w;
      }
      idx -= ex.groups[t];
    }
    return w;
  }
  if (wg >= m) {
    const int rows = (nblk - k - 2 + 1) / 2;  // group rows of the trailing part
    int idx = wg - m, gj = 0;
    while (gj < rows && idx >= rows - gj) {
      idx -= rows - gj;
      ++gj;
    }
    if (gj < rows) w = CholWork{1, k + 2 + 2 * (gj + idx), k + 2 + 2 * gj, k, 1, t_end};
    return w;
  }
  w = CholWork{0, k + 1 + (split == 2 ? 1 : 0) + wg, k + 1, k, 1, 0};
  return w;
}

// Cholesky launch k (k = -1 .. nblk - 2): workgroups 0 .. m - 1 own the next
// panel column, blocks (k + 1 + i, k + 1), and (when `apply`) first subtract
// panel k from it; the others apply panel k to the trailing columns k + 2 ..
// t_end - 1 (all rows below) in 2 x 2 groups of blocks, group column by group
// column, then run the extra super-panel groups of `x` (none: x.trail = -1).
// Columns from t_end on receive panel k later, with the rest of its
// super-panel (chol_trail_kernel, or the extra groups of a later launch).
// split = 0: every workgroup of the panel column factors the diagonal block
// itself (no launch waits for another). split = 1: only the diagonal block
// (one workgroup), which leaves its inverse in Dinv; split = 2: the blocks
// below it, which read that inverse, and the trailing part. Both forms do the
// same arithmetic in the same order.
__global__ __launch_bounds__(kThreads) void chol_step_kernel(float* L, float* Dinv, int n, int k, int t_end,
                                                            int apply, int split, int* status, int64_t ws,
                                                            CholExtra ex) {
  __shared__ __attribute__((aligned(16))) Tile tiles[6];
  __shared__ int bad;
  L = at_layer(L, ws, blockIdx.y);
  Dinv = at_layer(Dinv, ws, blockIdx.y);
  status = at_layer(status, ws, blockIdx.y);
  const int nblk = (n + kNb - 1) / kNb;
  const CholWork wk = chol_work_of((int)blockIdx.x, nblk, k, t_end, split, ex);
  if (wk.kind < 0) return;
  if (wk.kind == 1) {
    if (wk.np == 1) {
      trailing_2x2<1>(L, n, nblk, wk.p0, wk.R, wk.T, wk.t_end, tiles);
    } else {
      trailing_2x2<kLa>(L, n, nblk, wk.p0, wk.R, wk.T, wk.t_end, tiles);
    }
    return;
  }
  apply = apply && k >= 0;
  Tile &S = tiles[0], &M = tiles[1], &T = tiles[2], &U = tiles[3], &V = tiles[4], &P = tiles[5];
  const int r = wk.R, t = wk.T;  // block coordinates
  const int rr = min(kNb, n - r * kNb);
  float* Lrt = L + (int64_t)r * kNb * n + t * kNb;
  if (threadIdx.x == 0) bad = 0;

  // next panel column: updated diagonal block, factor, inverse
  const int d = k + 1;
  const int nd = min(kNb, n - d * kNb);
  const bool off = r != d;
  Frag fs, fv, ft, fu;
  if (split == 2) {
    // below the diagonal block: A_rd - L_rk L_dk^T (the quadrants as the
    // factor's other waves form them), then times the stored inverse
    if (apply) fetch(fv, L + (int64_t)d * kNb * n + k * kNb, n, nd, kNb);
    fetch(ft, Lrt, n, rr, nd);
    if (apply) fetch(fu, L + (int64_t)r * kNb * n + k * kNb, n, rr, kNb);
    fetch(fs, Dinv + (int64_t)d * kNb * kNb, kNb, kNb, kNb);
    if (apply) put(V, fv);
    put(P, ft);
    if (apply) put(U, fu);
    put(M, fs);
    __syncthreads();
    if (apply) {
      const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
      const int r0 = (wave >> 1) * 32, c0 = (wave & 1) * 32;
      f32x16 acc = {};
      mma<false, true>(acc, U, r0, 0, V, c0, 0, kNb, lane);
#pragma unroll
      for (int e = 0; e < 16; ++e) P[r0 + acc_row(e, lane)][c0 + (lane & 31)] -= acc[e];
      __syncthreads();
    }
    const f32x16 x = quad<false, true>(P, M);
    __syncthreads();
    quad_store(P, x, 1.f, false);
    __syncthreads();
    store_tile(P, Lrt, n, rr, nd);
    return;
  }
  fetch(fs, L + (int64_t)d * kNb * n + d * kNb, n, nd, nd);
  if (apply) fetch(fv, L + (int64_t)d * kNb * n + k * kNb, n, nd, kNb);
  if (off) {
    fetch(ft, Lrt, n, rr, nd);
    if (apply) fetch(fu, L + (int64_t)r * kNb * n + k * kNb, n, rr, kNb);
  }
  put(S, fs);
  if (apply) put(V, fv);
  if (off) {
    put(P, ft);
    if (apply) put(U, fu);
  }
  __syncthreads();
  if (apply) {
    quad_store(S, quad<false, true>(V, V), -1.f, true);
    __syncthreads();
  }
  // factor the diagonal block; an off-diagonal workgroup's other waves form
  // A_rd - L_rk L_dk^T meanwhile
  factor64(S, M, T, nd, &bad, off && apply ? &P : nullptr, &U, &V);
  if (!off) {
    store_tile(M, Dinv + (int64_t)d * kNb * kNb, kNb, kNb, kNb);
    if (threadIdx.x == 0 && bad) atomicOr(status, 1);
    return;
  }
  // L_rd = (A_rd - L_rk L_dk^T) . M^T
  const f32x16 x = quad<false, true>(P, M);
  __syncthreads();
  quad_store(P, x, 1.f, false);
  __syncthreads();
  store_tile(P, Lrt, n, rr, nd);
}

// ---------------------------------------------------------------- 256-block
// Triangular solves in block LDL^T form. With 256 x 256 diagonal blocks L_II of
// L, X_I = L_II^-1, Lh_rI = L_rI X_I (unit block-lower Lh, L = Lh diag(L_II)) and
// P_I = X_I^T X_I (the inverse of the I-th diagonal block of the Schur
// complements):
//   L Z = C      <=>  Lh Y = C,  Z_I = X_I Y_I
//   L^T dW = Z   <=>  Lh^T dW = V,  V_I = P_I Y_I
// Both unit-triangular sweeps are right-looking rank-256 GEMM updates with no
// diagonal work, one launch per block: Y_r -= Lh_rI Y_I (r > I) and
// dW_I -= Lh_JI^T dW_J (I < J). Lh overwrites the strictly-below-256-block part
// of L and its transpose is mirrored into the (otherwise zero) upper part, so
// that every GEMM operand is read as rows of a row-major matrix.
constexpr int kBb = 256;  // block size of the triangular sweeps
constexpr int kKc = 16;   // k rows per LDS chunk of the GEMM

// quad() accumulated into acc
template <bool TA, bool TB>
__device__ __forceinline__ void quad_acc(f32x16& acc, const Tile& A, const Tile& B) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  mma<TA, TB>(acc, A, (wave >> 1) * 32, 0, B, (wave & 1) * 32, 0, kNb, lane);
}
__device__ __forceinline__ void quad_put(Tile& D, const f32x16& acc, float sign) {
  quad_store(D, acc, sign, false);
}

// X_I = L_II^-1 for 256-block I = blockIdx.x, 64-column strip b = blockIdx.y:
// X_bb = Dinv_b and, for a > b, X_ab = -Dinv_a sum_{c=b}^{a-1} L_ac X_cb (64-block
// indices inside the 256-block). Writes the full 256 x 64 strip of X_I (zeros
// above the diagonal and in 64-blocks past the end of the matrix).
__global__ __launch_bounds__(kThreads) void inv256_kernel(const float* L, const float* Dinv, float* Xinv, int n,
                                                         int64_t ws) {
  __shared__ Tile Xc[4];
  __shared__ Tile U;
  L = at_layer(L, ws, blockIdx.z);
  Dinv = at_layer(Dinv, ws, blockIdx.z);
  Xinv = at_layer(Xinv, ws, blockIdx.z);
  const int nblk = (n + kNb - 1) / kNb;
  const int I = blockIdx.x, b = blockIdx.y;
  const int g0 = I * 4;                       // first 64-block of the 256-block
  const int n64 = min(4, nblk - g0);          // 64-blocks inside the matrix
  float* X = Xinv + (int64_t)I * kBb * kBb;  // [256][256], row-major
  if (b < n64) {
    load_tile(Xc[b], Dinv + (int64_t)(g0 + b) * kNb * kNb, kNb, kNb, kNb);
    __syncthreads();
    for (int a = b + 1; a < n64; ++a) {
      const int ra = min(kNb, n - (g0 + a) * kNb);
      f32x16 t = {};
      for (int c = b; c < a; ++c) {
        load_tile(U, L + (int64_t)(g0 + a) * kNb * n + (int64_t)(g0 + c) * kNb, n, ra, kNb);
        __syncthreads();
        quad_acc<false, false>(t, U, Xc[c]);
        __syncthreads();
      }
      // Xc[a] = -Dinv_a . T: T goes through Xc[a], Dinv_a through U
      quad_put(Xc[a], t, 1.f);
      load_tile(U, Dinv + (int64_t)(g0 + a) * kNb * kNb, kNb, kNb, kNb);
      __syncthreads();
      const f32x16 x = quad<false, false>(U, Xc[a]);
      __syncthreads();
      quad_put(Xc[a], x, -1.f);
      __syncthreads();
    }
  }
  for (int a = 0; a < 4; ++a) {
    float* dst = X + (int64_t)a * kNb * kBb + b * kNb;
    if (b < n64 && a >= b && a < n64) {
      store_tile(Xc[a], dst, kBb, kNb, kNb);
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int e = threadIdx.x + q * kThreads;
        const int r = e >> 4, c = (e & 15) * 4;
        *(f32x4*)(dst + (int64_t)r * kBb + c) = f32x4{0.f, 0.f, 0.f, 0.f};
      }
    }
  }
}

// Upper part of L from Lh: U[c][r] = L[r][c] for every (r, c) whose 256-block
// row is below its 256-block column. One 64 x 64 tile per workgroup.
__global__ __launch_bounds__(kThreads) void mirror_kernel(float* L, int n, int64_t ws) {
  __shared__ Tile T;
  L = at_layer(L, ws, blockIdx.y);
  const int nblk = (n + kNb - 1) / kNb;
  const int tr = blockIdx.x / nblk, tc = blockIdx.x % nblk;
  if (tr / 4 <= tc / 4) return;
  const int rr = min(kNb, n - tr * kNb), rc = min(kNb, n - tc * kNb);
  load_tile(T, L + (int64_t)tr * kNb * n + (int64_t)tc * kNb, n, rr, rc);
  __syncthreads();
  float* dst = L + (int64_t)tc * kNb * n + (int64_t)tr * kNb;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int e = threadIdx.x + q * kThreads;
    const int r = e >> 4, c = (e & 15) * 4;
    if (r < rc && c < rr) *(f32x4*)(dst + (int64_t)r * n + c) = f32x4{T[c][r], T[c + 1][r], T[c + 2][r], T[c + 3][r]};
  }
}

// C(m, n) = [C(m, n) -] sum_k A(m, k) B(k, n) for m < M, n < N, in fp32 MFMA.
// B(k, n) = B[k * ldb + n]. A(m, k) = A[k * lda + m] (k-major), or
// A[m * lda + k] for the m-major instantiation. One launch runs up to two jobs
// that share B, N and K (tiles of job 0 first), batched over blockIdx.y with
// element strides per batch and M growing by batch_dm per batch. Dimensions
// are multiples of 4 and rows 16-byte aligned. Operands are staged through
// LDS k-major (a row of 16 k-rows per chunk, double buffered) so that the
// 32 lanes of an MFMA operand read 32 consecutive floats.
struct GemmJob {
  const float* A;
  float* C;
  int M;
  int64_t lda, ldc;
  int sub;                    // 1: C -= A B, 0: C = A B
  const float* Cin = nullptr;  // with sub: read the minuend here instead of C (same ldc)
  int64_t la = 0, lc = 0;      // bytes per layer (blockIdx.z) of A and of C / Cin
  const float* B = nullptr;    // this job's own B operand and depth (gemm_ring_kernel only);
  int K = 0;                   // null / 0: the shared B and K below
};
struct GemmArgs {
  GemmJob job[2];
  int n_jobs;
  const float* B;
  int N, K;
  int64_t ldb;
  int64_t batch_a, batch_b, batch_c;
  int batch_dm;
  int64_t lb;  // bytes per layer (blockIdx.z) of B
};

template <int WM, int WN, int QM, int QN, bool A_MK>
__global__ __launch_bounds__(kThreads) void gemm_kernel(GemmArgs g) {
  constexpr int TM = WM * QM * 32, TN = WN * QN * 32;
  constexpr int SA = TM + 32, SB = TN + 32;  // row strides: the two k rows of an operand read sit 32 banks apart
  constexpr int kA4 = kKc * TM / 4;  // 16-byte pieces of an A chunk
  constexpr int NA = (kA4 + kThreads - 1) / kThreads, NB = kKc * TN / 4 / kThreads;
  static_assert(WM * WN == kThreads / 64 && NB >= 1 && kA4 % 64 == 0, "tile shape");
  __shared__ __attribute__((aligned(16))) float As[2][kKc][SA];
  __shared__ __attribute__((aligned(16))) float Bs[2][kKc][SB];

  const int tiles_n = (g.N + TN - 1) / TN;
  const int dm = (int)blockIdx.y * g.batch_dm;
  const int m_tiles0 = (g.job[0].M + dm + TM - 1) / TM;
  int t = blockIdx.x;
  const bool second = t >= m_tiles0 * tiles_n;
  if (second) {
    if (g.n_jobs < 2) return;
    t -= m_tiles0 * tiles_n;
  }
  const float* A = second ? g.job[1].A : g.job[0].A;
  float* C = second ? g.job[1].C : g.job[0].C;
  const int M = (second ? g.job[1].M : g.job[0].M) + dm;
  const int64_t lda = second ? g.job[1].lda : g.job[0].lda;
  const int64_t ldc = second ? g.job[1].ldc : g.job[0].ldc;
  const int sub = second ? g.job[1].sub : g.job[0].sub;
  const int m0 = (t / tiles_n) * TM, n0 = (t % tiles_n) * TN;
  if (m0 >= M) return;
  const int layer = blockIdx.z;
  A = at_layer(A, second ? g.job[1].la : g.job[0].la, layer) + blockIdx.y * g.batch_a;
  const float* B = at_layer(g.B, g.lb, layer) + blockIdx.y * g.batch_b;
  C = at_layer(C, second ? g.job[1].lc : g.job[0].lc, layer) + blockIdx.y * g.batch_c;
  const int N = g.N, K = g.K;

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int h = lane >> 5, l32 = lane & 31;
  const int wm0 = (wave / WN) * QM * 32, wn0 = (wave % WN) * QN * 32;

  f32x4 ra[NA], rb[NB];
  auto fetch_chunk = [&](int k0) {
#pragma unroll
    for (int q = 0; q < NA; ++q) {
      const int e = threadIdx.x + q * kThreads;
      if (e >= kA4) break;  // (wave-uniform: kA4 is a multiple of 64)
      if (A_MK) {
        const int m = e / (kKc / 4), k = (e % (kKc / 4)) * 4;
        ra[q] = (m0 + m < M && k0 + k < K) ? *(const f32x4*)(A + (int64_t)(m0 + m) * lda + k0 + k)
                                             : f32x4{0.f, 0.f, 0.f, 0.f};
      } else {
        const int k = e / (TM / 4), m = (e % (TM / 4)) * 4;
        ra[q] = (k0 + k < K && m0 + m < M) ? *(const f32x4*)(A + (int64_t)(k0 + k) * lda + m0 + m)
                                             : f32x4{0.f, 0.f, 0.f, 0.f};
      }
    }
#pragma unroll
    for (int q = 0; q < NB; ++q) {
      const int e = threadIdx.x + q * kThreads;
      const int k = e / (TN / 4), nn = (e % (TN / 4)) * 4;
      rb[q] = (k0 + k < K && n0 + nn < N) ? *(const f32x4*)(B + (int64_t)(k0 + k) * g.ldb + n0 + nn)
                                            : f32x4{0.f, 0.f, 0.f, 0.f};
    }
  };
  auto put_chunk = [&](int buf) {
#pragma unroll
    for (int q = 0; q < NA; ++q) {
      const int e = threadIdx.x + q * kThreads;
      if (e >= kA4) break;
      if (A_MK) {
        const int m = e / (kKc / 4), k = (e % (kKc / 4)) * 4;
#pragma unroll
        for (int j = 0; j < 4; ++j) As[buf][k + j][m] = ra[q][j];
      } else {
        const int k = e / (TM / 4), m = (e % (TM / 4)) * 4;
        *(f32x4*)&As[buf][k][m] = ra[q];
      }
    }
#pragma unroll
    for (int q = 0; q < NB; ++q) {
      const int e = threadIdx.x + q * kThreads;
      const int k = e / (TN / 4), nn = (e % (TN / 4)) * 4;
      *(f32x4*)&Bs[buf][k][nn] = rb[q];
    }
  };

  f32x16 acc[QM][QN];
#pragma unroll
  for (int i = 0; i < QM; ++i)
#pragma unroll
    for (int j = 0; j < QN; ++j) acc[i][j] = f32x16{};

  const int nk = (K + kKc - 1) / kKc;
  fetch_chunk(0);
  put_chunk(0);
  __syncthreads();
  for (int c = 0; c < nk; ++c) {
    const int buf = c & 1;
    if (c + 1 < nk) fetch_chunk((c + 1) * kKc);
#pragma unroll
    for (int kk = 0; kk < kKc; kk += 2) {
      float a[QM], b[QN];
#pragma unroll
      for (int i = 0; i < QM; ++i) a[i] = As[buf][kk + h][wm0 + 32 * i + l32];
#pragma unroll
      for (int j = 0; j < QN; ++j) b[j] = Bs[buf][kk + h][wn0 + 32 * j + l32];
#pragma unroll
      for (int i = 0; i < QM; ++i)
#pragma unroll
        for (int j = 0; j < QN; ++j) acc[i][j] = mfma_f32(a[i], b[j], acc[i][j]);
    }
    if (c + 1 < nk) put_chunk(buf ^ 1);
    __syncthreads();
  }

#pragma unroll
  for (int i = 0; i < QM; ++i)
#pragma unroll
    for (int j = 0; j < QN; ++j) {
      const int col = n0 + wn0 + 32 * j + l32;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + wm0 + 32 * i + acc_row(r, lane);
        if (row < M && col < N) {
          float* p = C + (int64_t)row * ldc + col;
          *p = sub ? *p - acc[i][j][r] : acc[i][j][r];
        }
      }
    }
}

// <dW, C> and ||dW||^2 in two passes: each of kEpsBlocks workgroups reduces a
// grid-strided share (16-byte loads, n a multiple of 4) to one pair in
// part[2 * block], then a single workgroup adds the pairs into scalars[0], [1].
constexpr int kEpsBlocks = 512;
__device__ __forceinline__ void block_sum2(double& a, double& b, double (*red)[kThreads / 64]) {
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
  a = 0;
  b = 0;
  for (int w = 0; w < kThreads / 64; ++w) {
    a += red[0][w];
    b += red[1][w];
  }
}
__global__ __launch_bounds__(kThreads) void eps_partial_kernel(const float* dw, const float* C, int64_t n,
                                                               double* part, int64_t ws, int64_t dws) {
  __shared__ double red[2][kThreads / 64];
  dw = at_layer(dw, dws, blockIdx.y);
  C = at_layer(C, ws, blockIdx.y);
  part = at_layer(part, ws, blockIdx.y);
  double a = 0, b = 0;
  const int64_t n4 = n / 4;
  for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n4; i += (int64_t)gridDim.x * kThreads) {
    const f32x4 w = *(const f32x4*)(dw + 4 * i);
    const f32x4 c = *(const f32x4*)(C + 4 * i);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      a += (double)w[j] * (double)c[j];
      b += (double)w[j] * (double)w[j];
    }
  }
  block_sum2(a, b, red);
  if (threadIdx.x == 0) {
    part[2 * blockIdx.x] = a;
    part[2 * blockIdx.x + 1] = b;
  }
}
// sc: [0] s = sum ||R||^2 (from the statistics), then written here: [2] <dW, C>,
// [3] ||dW||^2, [4] eps = s - <dW, C> - lambda ||dW||^2 (Eq. 6; each operation
// rounded on its own), [5] the status word as a double. eps_out / status_out,
// when given, receive eps and the status word as well.
__global__ __launch_bounds__(kThreads) void eps_final_kernel(const double* part, int n_part, double* sc,
                                                             double lambda, const int* status, double* eps_out,
                                                             int* status_out, int64_t ws) {
  __shared__ double red[2][kThreads / 64];
  const int layer = blockIdx.y;
  part = at_layer(part, ws, layer);
  sc = at_layer(sc, ws, layer);
  status = at_layer(status, ws, layer);
  double a = 0, b = 0;
  for (int i = threadIdx.x; i < n_part; i += kThreads) {
    a += part[2 * i];
    b += part[2 * i + 1];
  }
  block_sum2(a, b, red);
  if (threadIdx.x == 0) {
    const double e = __dsub_rn(__dsub_rn(sc[0], a), __dmul_rn(lambda, b));
    const int st = *status;
    sc[2] = a;
    sc[3] = b;
    sc[4] = e;
    sc[5] = (double)st;
    if (eps_out) eps_out[layer] = e;
    if (status_out) status_out[layer] = st;
  }
}

}  // namespace

namespace {

// ---------------------------------------------------------------- ring GEMM
// The sweeps' GEMM (both operands k-major: A(m, k) = A[k * lda + m]) with the
// operands staged HBM -> LDS by buffer loads straight into LDS, in a ring of 4
// stages of 16 k-rows, 3 stages ahead of the MFMAs. A stage side holds 16 rows
// of the tile's TM (or TN) columns, 16-byte chunk c of row k stored at chunk
// c ^ 8 (k & 1): the two k-rows read by one MFMA operand sit 32 banks apart.
// The buffer descriptor of a side ends at the last valid element of the job,
// so k-rows past K read as zero; columns past M or N read finite neighbouring
// data that only reaches outputs that are not stored.
constexpr int kRing = 4;

template <int N>
__device__ __forceinline__ void vm_wait() {
  static_assert(N >= 0 && N <= 63, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"i"(N) : "memory");
}

template <int T>
__device__ __forceinline__ void ring_side(const float* src, int64_t ld, int k0, int kend, int c0, int cend, char* dst,
                                          int wave, int lane) {
  int64_t nrec = ((int64_t)(kend - k0 - 1) * ld + (cend - c0)) * 4;
  if (nrec < 0) nrec = 0;
  if (nrec > 0x7fffffff) nrec = 0x7fffffff;
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(src + (int64_t)k0 * ld + c0), 0, (int)nrec, 0x00020000);
  constexpr int kChunks = T / 4;  // 16-byte chunks per row
#pragma unroll
  for (int q = 0; q < kKc * T * 4 / (kThreads * 16); ++q) {
    const int slot = (q * 4 + wave) * 64 + lane;
    const int row = slot / kChunks;
    const int c = (slot % kChunks) ^ ((row & 1) << 3);
    const int voff = (int)((row * ld + c * 4) * 4);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (ISPA_LDS void*)(dst + (q * 4 + wave) * 1024), 16, voff, 0, 0, 0);
  }
}

template <int QM, int QN>
struct RingRegs {
  float a[2][QM], b[2][QN];
};

// LDS reads of k-row pair KK of stage buffer BUF into register set S
template <int IMMA, int IMMB, int QM, int QN>
__device__ __forceinline__ void ring_issue(const uint32_t (&oa)[QM], const uint32_t (&ob)[QN], float (&a)[QM],
                                           float (&b)[QN]) {
#pragma unroll
  for (int i = 0; i < QM; ++i) asm volatile("ds_read_b32 %0, %1 offset:%2" : "=v"(a[i]) : "v"(oa[i]), "i"(IMMA));
#pragma unroll
  for (int j = 0; j < QN; ++j) asm volatile("ds_read_b32 %0, %1 offset:%2" : "=v"(b[j]) : "v"(ob[j]), "i"(IMMB));
}

// at most N LDS operations outstanding: the reads into a, b have landed
template <int N, int QM, int QN>
__device__ __forceinline__ void ring_wait(float (&a)[QM], float (&b)[QN]) {
  static_assert(N >= 0 && N <= 15 && ((QM == 2 && QN == 2) || (QM == 1 && QN == 1)), "shape");
  if constexpr (QM == 2) {
    asm volatile("s_waitcnt lgkmcnt(%4)" : "+v"(a[0]), "+v"(a[1]), "+v"(b[0]), "+v"(b[1]) : "i"(N));
  } else {
    asm volatile("s_waitcnt lgkmcnt(%2)" : "+v"(a[0]), "+v"(b[0]) : "i"(N));
  }
}

template <int BUF, int KK, int TM, int TN, int QM, int QN>
__device__ __forceinline__ void ring_ksteps(const uint32_t (&oa)[QM], const uint32_t (&ob)[QN], RingRegs<QM, QN>& r,
                                            f32x16 (&acc)[QM][QN]) {
  constexpr int kStage = kKc * (TM + TN) * 4;
  constexpr int cur = (KK / 2) & 1;
  if constexpr (KK + 2 < kKc) {
    ring_issue<BUF * kStage + (KK + 2) * TM * 4, BUF * kStage + (KK + 2) * TN * 4, QM, QN>(oa, ob, r.a[cur ^ 1],
                                                                                           r.b[cur ^ 1]);
    ring_wait<QM + QN, QM, QN>(r.a[cur], r.b[cur]);
  } else {
    ring_wait<0, QM, QN>(r.a[cur], r.b[cur]);
  }
#pragma unroll
  for (int i = 0; i < QM; ++i)
#pragma unroll
    for (int j = 0; j < QN; ++j) acc[i][j] = mfma_f32(r.a[cur][i], r.b[cur][j], acc[i][j]);
  if constexpr (KK + 2 < kKc) ring_ksteps<BUF, KK + 2, TM, TN, QM, QN>(oa, ob, r, acc);
}

struct RingTile {
  const float* A;
  const float* B;
  int64_t lda, ldb;
  int M, N, K, m0, n0, steps, wave, lane;
};

template <int TM, int TN>
__device__ __forceinline__ void ring_load(const RingTile& t, char* smem, int s) {
  constexpr int kStage = kKc * (TM + TN) * 4;
  char* d = smem + (s % kRing) * kStage;
  const int k0 = s * kKc;
  ring_side<TM>(t.A, t.lda, k0, t.K, t.m0, t.M, d, t.wave, t.lane);
  ring_side<TN>(t.B, t.ldb, k0, t.K, t.n0, t.N, d + kKc * TM * 4, t.wave, t.lane);
}

// stage s from ring buffer BUF = s % 4: loads of stage s + 3, the MFMAs of s,
// then wait for stage s + 1 (direct loads retire in order) and synchronise
template <int BUF, int TM, int TN, int QM, int QN>
__device__ __forceinline__ void ring_stage(const RingTile& t, char* smem, const uint32_t (&oa)[QM],
                                           const uint32_t (&ob)[QN], f32x16 (&acc)[QM][QN], int s) {
  constexpr int kLoads = (TM + TN) / 64;  // direct loads per thread per stage
  if (s + 3 < t.steps) ring_load<TM, TN>(t, smem, s + 3);
  RingRegs<QM, QN> r;
  ring_issue<BUF * kKc * (TM + TN) * 4, BUF * kKc * (TM + TN) * 4, QM, QN>(oa, ob, r.a[0], r.b[0]);
  ring_ksteps<BUF, 0, TM, TN, QM, QN>(oa, ob, r, acc);
  const int younger = t.steps - (s + 2);
  if (younger >= 2) {
    vm_wait<2 * kLoads>();
  } else if (younger == 1) {
    vm_wait<kLoads>();
  } else {
    vm_wait<0>();
  }
  // the direct loads of stage s + 1 have landed (vmcnt above) and every LDS
  // read of this wave has completed (lgkmcnt(0) in the last k-step): a bare barrier
  // suffices, where a fenced one would also wait for the younger stages
  __builtin_amdgcn_s_barrier();
}

template <int WM, int WN, int QM, int QN>
__global__ __launch_bounds__(kThreads) void gemm_ring_kernel(GemmArgs g) {
  constexpr int TM = WM * QM * 32, TN = WN * QN * 32;
  constexpr int kLoads = (TM + TN) / 64;
  static_assert(WM * WN == kThreads / 64, "4 waves");
  __shared__ __attribute__((aligned(1024))) char smem[kRing * kKc * (TM + TN) * 4];

  const int tiles_n = (g.N + TN - 1) / TN;
  const int m_tiles0 = (g.job[0].M + TM - 1) / TM;
  int tt = blockIdx.x;
  const bool second = tt >= m_tiles0 * tiles_n;
  if (second) {
    if (g.n_jobs < 2) return;
    tt -= m_tiles0 * tiles_n;
  }
  RingTile t;
  t.A = second ? g.job[1].A : g.job[0].A;
  float* C = second ? g.job[1].C : g.job[0].C;
  t.M = second ? g.job[1].M : g.job[0].M;
  t.lda = second ? g.job[1].lda : g.job[0].lda;
  const int64_t ldc = second ? g.job[1].ldc : g.job[0].ldc;
  const int sub = second ? g.job[1].sub : g.job[0].sub;
  const float* Cin = second ? g.job[1].Cin : g.job[0].Cin;
  if (Cin == nullptr) Cin = C;
  t.m0 = (tt / tiles_n) * TM;
  t.n0 = (tt % tiles_n) * TN;
  if (t.m0 >= t.M) return;
  {
    const int layer = blockIdx.z;
    const int64_t lc = second ? g.job[1].lc : g.job[0].lc;
    t.A = at_layer(t.A, second ? g.job[1].la : g.job[0].la, layer);
    C = at_layer(C, lc, layer);
    Cin = at_layer(Cin, lc, layer);
  }
  {
    const GemmJob& jb = second ? g.job[1] : g.job[0];
    t.B = at_layer(jb.B ? jb.B : g.B, g.lb, blockIdx.z);
    t.K = jb.K ? jb.K : g.K;
  }
  t.ldb = g.ldb;
  t.N = g.N;
  t.steps = (t.K + kKc - 1) / kKc;
  t.lane = threadIdx.x & 63;
  t.wave = threadIdx.x >> 6;
  const int h = t.lane >> 5, l32 = t.lane & 31;
  const int wm0 = (t.wave / WN) * QM * 32, wn0 = (t.wave % WN) * QN * 32;

  const uint32_t lds0 = (uint32_t)(uintptr_t)(ISPA_LDS const void*)smem;
  uint32_t oa[QM], ob[QN];
#pragma unroll
  for (int i = 0; i < QM; ++i) oa[i] = lds0 + h * TM * 4 + (((wm0 + 32 * i + l32) ^ (32 * h)) << 2);
#pragma unroll
  for (int j = 0; j < QN; ++j) ob[j] = lds0 + kKc * TM * 4 + h * TN * 4 + (((wn0 + 32 * j + l32) ^ (32 * h)) << 2);

  f32x16 acc[QM][QN];
#pragma unroll
  for (int i = 0; i < QM; ++i)
#pragma unroll
    for (int j = 0; j < QN; ++j) acc[i][j] = f32x16{};

  for (int s = 0; s < 3 && s < t.steps; ++s) ring_load<TM, TN>(t, smem, s);
  if (t.steps >= 3) {
    vm_wait<2 * kLoads>();
  } else if (t.steps == 2) {
    vm_wait<kLoads>();
  } else {
    vm_wait<0>();
  }
  __builtin_amdgcn_s_barrier();  // stage 0 has landed (vmcnt above)
  for (int s = 0; s < t.steps; s += kRing) {
    ring_stage<0, TM, TN, QM, QN>(t, smem, oa, ob, acc, s);
    if (s + 1 < t.steps) ring_stage<1, TM, TN, QM, QN>(t, smem, oa, ob, acc, s + 1);
    if (s + 2 < t.steps) ring_stage<2, TM, TN, QM, QN>(t, smem, oa, ob, acc, s + 2);
    if (s + 3 < t.steps) ring_stage<3, TM, TN, QM, QN>(t, smem, oa, ob, acc, s + 3);
  }

  const int lane = t.lane;
#pragma unroll
  for (int i = 0; i < QM; ++i)
#pragma unroll
    for (int j = 0; j < QN; ++j) {
      const int col = t.n0 + wn0 + 32 * j + l32;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = t.m0 + wm0 + 32 * i + acc_row(r, lane);
        if (row < t.M && col < t.N) {
          const int64_t o = (int64_t)row * ldc + col;
          C[o] = sub ? Cin[o] - acc[i][j][r] : acc[i][j][r];
        }
      }
    }
}

}  // namespace

// Dinv: 64 x 64 inverses of the diagonal blocks of L, then X_I and P_I of the
// 256-blocks.
size_t solve_dinv_bytes(int d) {
  const int nblk = (d + kNb - 1) / kNb;
  const int nb = (d + kBb - 1) / kBb;
  return (size_t)nblk * kNb * kNb * sizeof(float) + 2 * (size_t)nb * kBb * kBb * sizeof(float);
}

namespace {

// Launches C (-)= A B over 64 x 64 output tiles, for `layers` layers.
hipError_t launch_gemm(const GemmArgs& g, int layers, hipStream_t stream) {
  int tiles = 0;
  for (int j = 0; j < g.n_jobs; ++j) tiles += ((g.job[j].M + 63) / 64) * ((g.N + 63) / 64);
  // 64 x 64 tiles at every size: 32 KB of LDS, so several workgroups share a CU
  // and hide each other's load latency, and the last round is finely grained
  // (measured against 128 x 128 and 128 x 64 tiles: the 5120-row solve takes
  // 5.1 ms with 64 x 64 tiles throughout, 6.2 ms with 128 x 128)
  hipLaunchKernelGGL((gemm_ring_kernel<2, 2, 1, 1>), dim3(tiles, 1, layers), dim3(kThreads), 0, stream, g);
  return hipGetLastError();
}

}  // namespace

// A second stream per device for one half of the sweeps' columns, with the
// events of the fork and the join (created once, kept for the process), from
// d = kSweepTwoFrom on; ISPA_SOLVE_TWO_STREAMS=0 / 1 switches it off / on at
// every size with at least two column tiles.
namespace {
constexpr int kSweepCols = 64;  // the halves split at a multiple of the tile width
constexpr int kSweepTwoFrom = 4096;  // smallest d whose sweeps go on two streams
struct SideStream {
  hipStream_t s = nullptr;
  hipEvent_t fork = nullptr, join = nullptr;
  bool tried = false;
};
std::mutex g_side_mu;
SideStream g_side[64];

SideStream* side_stream(int d) {
  const char* env = getenv("ISPA_SOLVE_TWO_STREAMS");
  if (env != nullptr ? env[0] != '1' : d < kSweepTwoFrom) return nullptr;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
  std::lock_guard<std::mutex> lock(g_side_mu);
  SideStream& t = g_side[dev];
  if (!t.tried) {
    t.tried = true;
    if (hipStreamCreateWithFlags(&t.s, hipStreamNonBlocking) != hipSuccess ||
        hipEventCreateWithFlags(&t.fork, hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&t.join, hipEventDisableTiming) != hipSuccess)
      t.s = nullptr;
  }
  return t.s != nullptr ? &t : nullptr;
}
}  // namespace

// The launches of a single layer's look-ahead factorisation (launch k at
// index k + 1): its workgroups, its t_end and its extra tasks (see launch_solve).
struct LookaheadPlan {
  std::vector<int> grid, t_end;
  std::vector<CholExtra> extra;
};
static void lookahead_plan(int nblk, int n_cu, LookaheadPlan* plan) {
  plan->grid.assign(nblk, 0);
  plan->t_end.assign(nblk, 0);
  plan->extra.assign(nblk, CholExtra{});
  int next_sp[kMaxTasks] = {};               // per band: the next group it receives
  const int n_bands = (nblk - 2) / kLa + 1;  // bands 1 .. n_bands - 1 start inside the matrix
  auto band_groups = [&](int b) {
    int g = 0;
    for (int T = b * kLa + 1; T < min(nblk, b * kLa + kLa + 1); T += 2) g += (nblk - T + 1) / 2;
    return g;
  };
  for (int k = -1; k <= nblk - 2; ++k) {
    const int m = nblk - 1 - k;
    const int t_end = k >= 0 ? min(nblk, k / kLa * kLa + kLa + 1) : 0;
    const int rows = (nblk - k - 2 + 1) / 2;
    const int cols = k >= 0 && t_end > k + 2 ? (t_end - k - 2 + 1) / 2 : 0;
    CholExtra x;
    memset(&x, 0, sizeof(x));
    x.trail = cols * rows - cols * (cols - 1) / 2;
    int cand[kMaxTasks][3], n_cand = 0;  // deadline, band, group
    for (int b = 1; b < n_bands; ++b) {
      const int sp = next_sp[b];
      if (sp <= b - 1 && k >= sp * kLa + kLa - 1) {
        cand[n_cand][0] = sp == b - 1 ? kLa * b - 1 : (kLa - 1) * b + sp;
        cand[n_cand][1] = b;
        cand[n_cand][2] = sp;
        ++n_cand;
      }
    }
    for (int i = 1; i < n_cand; ++i)  // by deadline, then band
      for (int j = i; j > 0 && (cand[j][0] < cand[j - 1][0] ||
                                (cand[j][0] == cand[j - 1][0] && cand[j][1] < cand[j - 1][1])); --j)
        for (int f = 0; f < 3; ++f) std::swap(cand[j][f], cand[j - 1][f]);
    // the rounds of workgroups the launch needs for its due tasks, filled up
    int used = m + x.trail, due = used;
    for (int i = 0; i < n_cand; ++i)
      if (cand[i][0] == k) due += band_groups(cand[i][1]);
    const int cap = (due + n_cu - 1) / n_cu * n_cu;
    for (int i = 0; i < n_cand; ++i) {
      const int b = cand[i][1];
      const int g = band_groups(b);
      if (cand[i][0] == k || used + g <= cap) {
        x.band[x.n_tasks] = b;
        x.sp[x.n_tasks] = cand[i][2];
        x.groups[x.n_tasks] = g;
        ++x.n_tasks;
        used += g;
        ++next_sp[b];
      }
    }
    plan->grid[k + 1] = used;
    plan->t_end[k + 1] = t_end;
    plan->extra[k + 1] = x;
  }
}

int solve_lookahead_check(int nblk, int n_cu) {
  if (nblk < 1 || (nblk - 2) / kLa + 1 >= kMaxTasks || n_cu < 1) return -1;
  LookaheadPlan plan;
  lookahead_plan(nblk, n_cu, &plan);
  // per block (r, c), r >= c: the next panel it must receive, and the last
  // launch that wrote it
  std::vector<int> next((size_t)nblk * nblk, 0), stamp((size_t)nblk * nblk, -2);
  for (int k = -1; k <= nblk - 2; ++k) {
    const int fail = k + 2;
    auto receive = [&](int r, int c, int p0, int np) {
      if (r < c || r >= nblk || c >= nblk) return false;
      const size_t b = (size_t)r * nblk + c;
      if (stamp[b] == k) return false;  // written twice in one launch
      stamp[b] = k;
      for (int p = p0; p < p0 + np; ++p) {
        // in panel order, panel p factored already (by launch p - 1), left of c
        if (p != next[b] || p > k || p >= c) return false;
        ++next[b];
      }
      return true;
    };
    for (int wg = 0; wg < plan.grid[k + 1]; ++wg) {
      const CholWork w = chol_work_of(wg, nblk, k, plan.t_end[k + 1], 0, plan.extra[k + 1]);
      if (w.kind == 0) {
        if (!receive(w.R, w.T, k, k >= 0 ? 1 : 0)) return fail;
      } else if (w.kind == 1) {
        for (int i = 0; i < 4; ++i) {
          const int br = w.R + i / 2, bc = w.T + i % 2;
          if (br < nblk && bc <= br && bc < w.t_end && !receive(br, bc, w.p0, w.np)) return fail;
        }
      }
    }
    // the launch has factored column k + 1: every block of it complete
    for (int r = k + 1; r < nblk; ++r)
      if (next[(size_t)r * nblk + k + 1] != k + 1) return fail;
  }
  for (int r = 0; r < nblk; ++r)
    for (int c = 0; c <= r; ++c)
      if (next[(size_t)r * nblk + c] != c) return nblk + 1;
  return 0;
}

// A single layer's factorisation in the look-ahead form (below) from 48
// panels on (measured: 80 panels 5.07 -> 4.74 ms per solve, 48 panels 1.76 ->
// 1.70 ms, 24 panels 0.654 -> 0.656 ms); ISPA_SOLVE_LOOKAHEAD=0 / 1 switches
// it off / on at every size.
static bool solve_lookahead(int nblk) {
  if ((nblk - 2) / kLa + 1 >= kMaxTasks) return false;  // bands beyond the task table
  const char* env = getenv("ISPA_SOLVE_LOOKAHEAD");
  if (env != nullptr) return env[0] == '1';
  return nblk >= 48;
}

hipError_t launch_solve(const float* G, const float* C, int d, int d_out, float lambda, float* delta_w,
                        const SolveWork& w, hipStream_t stream) {
  const int nblk = (d + kNb - 1) / kNb;
  const int nb = (d + kBb - 1) / kBb;
  float* xinv = w.dinv + (size_t)nblk * kNb * kNb;  // [nb][256][256]
  float* pinv = xinv + (size_t)nb * kBb * kBb;       // [nb][256][256]
  float* L = w.L;
  float* Y = w.work;
  // layers: workspaces (G, C, L, Y, the inverses, status, scalars) `ws` bytes
  // apart, the layers' dW `dws` bytes apart
  const int nl = w.n_layers;
  const int64_t ws = w.ws_stride, dws = w.dw_stride;
  hipLaunchKernelGGL(solve_init_kernel, dim3(d, nl), dim3(256), 0, stream, G, L, d, lambda, w.status, ws);
  // Several layers: the panels are grouped kSup at a time (super-panels);
  // launch k applies panel k only to the columns of its own super-panel, and
  // the rest of the trailing triangle receives the super-panel's panels
  // together, in one launch that keeps each block in registers across them,
  // once its last panel is factored (a quarter of the trailing-matrix traffic
  // of applying each panel everywhere; the same arithmetic in the same order).
  // A single layer's factorisation is a chain of launches bound by their
  // latency, to which an extra launch per super-panel would add: it takes the
  // look-ahead form below from 48 panels on, and below that applies every
  // panel everywhere at once.
  const int sup = kSup;
  CholExtra none;
  memset(&none, 0, sizeof(none));
  none.trail = -1;
  if (nl == 1 && solve_lookahead(nblk)) {
    // Look-ahead form (one layer), with the panels in groups of kLa = 2: launch k
    // applies panel k only up to block column 2 s + 2, s = k / 2 its group (the
    // rest of the group and the first column of the next). The other columns
    // receive whole groups in tasks (band, group) that ride along as extra
    // workgroups in the panel launches: task (b, s) can run once panel 2 s + 1
    // is factored (launch 2 s + 1 on), after task (b, s - 1), and must be done
    // before launch 2 b applies panel 2 b to band b, so (b, b - 1) runs in
    // launch 2 b - 1 and (b, s < b - 1) by launch b + s. Each launch takes
    // every task whose deadline it is, then more of its available tasks,
    // earliest deadline first, as many as fill the rounds of workgroups on
    // the chip that the launch needs anyway (one at least). A task's
    // workgroup (two panels on a 2 x 2 group of blocks, ~18.5 us) takes a
    // little longer than the launch's panel chain (~15.5 us); with groups of
    // four panels it took ~26 us (at 80 panels: 4.93 ms per solve, against
    // 4.74 ms with groups of two and 5.07 ms without look-ahead). Each block
    // still receives every panel once, in panel order, with the same
    // arithmetic: bit for bit the factor of the other forms.
    const int n_cu = attn_cu_count() > 0 ? attn_cu_count() : 256;
    LookaheadPlan plan;
    lookahead_plan(nblk, n_cu, &plan);
    for (int k = -1; k <= nblk - 2; ++k)
      hipLaunchKernelGGL(chol_step_kernel, dim3(plan.grid[k + 1], 1), dim3(kThreads), 0, stream, L, w.dinv, d, k,
                         plan.t_end[k + 1], k >= 0 ? 1 : 0, 0, w.status, ws, plan.extra[k + 1]);
  } else {
    const int c_def = nl > 1 ? nblk + sup : 0;
    for (int k = -1; k <= nblk - 2; ++k) {
      const int c = k + 1;                          // the panel column this launch factors
      int apply = k >= 0 ? 1 : 0;
      int t_end;
      if (c > c_def) {
        t_end = nblk;
      } else if (c % sup == 0) {
        if (c > 0) {
          const int gr = (nblk - c + 1) / 2;
          hipLaunchKernelGGL(chol_trail_kernel, dim3(gr * (gr + 1) / 2, nl), dim3(kThreads), 0, stream, L, d,
                             c - sup, c, ws);
        }
        apply = 0;                                  // panel k reached column c with its super-panel
        t_end = c;                                  // and no column of its super-panel is left
      } else {
        t_end = min(nblk, (c / sup + 1) * sup);
      }
      const int m = nblk - 1 - k;                   // blocks of the next panel column
      const int rows = (nblk - k - 2 + 1) / 2;      // group rows of the trailing part
      const int cols = k >= 0 && t_end > k + 2 ? (t_end - k - 2 + 1) / 2 : 0;  // launch -1 has no panel to apply
      const int groups = cols * rows - cols * (cols - 1) / 2;
      if (nl == 1) {
        hipLaunchKernelGGL(chol_step_kernel, dim3(m + groups, nl), dim3(kThreads), 0, stream, L, w.dinv, d, k, t_end,
                           apply, 0, w.status, ws, none);
      } else {
        // with many layers the diagonal block is factored once per layer, in its
        // own launch, rather than once per block of the column
        hipLaunchKernelGGL(chol_step_kernel, dim3(1, nl), dim3(kThreads), 0, stream, L, w.dinv, d, k, t_end, apply, 1,
                           w.status, ws, none);
        if (m - 1 + groups > 0)
          hipLaunchKernelGGL(chol_step_kernel, dim3(m - 1 + groups, nl), dim3(kThreads), 0, stream, L, w.dinv, d, k,
                             t_end, apply, 2, w.status, ws, none);
      }
    }
  }
  // X_I, P_I = X_I^T X_I, Lh below the 256-block diagonal, its mirror above
  hipLaunchKernelGGL(inv256_kernel, dim3(nb, 4, nl), dim3(kThreads), 0, stream, L, w.dinv, xinv, d, ws);
  {
    GemmArgs g = {};
    g.job[0] = GemmJob{xinv, pinv, kBb, kBb, kBb, 0};
    g.job[0].la = g.job[0].lc = ws;
    g.lb = ws;
    g.n_jobs = 1;
    g.B = xinv;
    g.N = kBb;
    g.K = kBb;
    g.ldb = kBb;
    g.batch_a = g.batch_b = g.batch_c = (int64_t)kBb * kBb;
    hipLaunchKernelGGL((gemm_kernel<2, 2, 1, 1, false>), dim3(16, nb, nl), dim3(kThreads), 0, stream, g);
  }
  if (nb > 1) {
    // Lh_rI = L_rI X_I in place: a workgroup owns 32 rows x the whole 256-block
    // (all of its A is read before any of its C is written)
    GemmArgs g = {};
    float* first = L + (int64_t)kBb * d;  // rows of block 1, columns of block 0
    g.job[0] = GemmJob{first, first, d - kBb, d, d, 0};
    g.job[0].la = g.job[0].lc = ws;
    g.lb = ws;
    g.n_jobs = 1;
    g.B = xinv;
    g.N = kBb;
    g.K = kBb;
    g.ldb = kBb;
    g.batch_a = g.batch_c = (int64_t)kBb * d + kBb;
    g.batch_b = (int64_t)kBb * kBb;
    g.batch_dm = -kBb;
    hipLaunchKernelGGL((gemm_kernel<1, 4, 1, 2, true>), dim3((d - kBb + 31) / 32, nb - 1, nl), dim3(kThreads), 0,
                       stream, g);
    hipLaunchKernelGGL(mirror_kernel, dim3(nblk * nblk, nl), dim3(kThreads), 0, stream, L, d, ws);
  }
  // The sweeps treat each column of the right-hand side on its own, so from
  // d = 4096 on the columns go in two halves, each on a stream of its own (the
  // caller's and a second one), whose launches fill each other's last rounds
  // of tiles and hide each other's short launches; every element's arithmetic
  // is unchanged. Measured (one solve, alternating, medians of 10): d = 5120
  // 4.75 -> 4.59 ms; d = 3072 1.70 -> 1.72, 2560 1.30 -> 1.34, 2048 0.91 ->
  // 0.97, 1536 0.66 -> 0.69 ms (halves too small to fill the chip).
  auto yblk = [&](auto* base, int I) { return base + (int64_t)I * kBb * d_out; };
  auto kblk = [&](int I) { return min(kBb, d - I * kBb); };
  auto lup = [&](int I, int r) { return L + (int64_t)I * kBb * d + (int64_t)r * kBb; };  // rows of I, columns of r
  auto sweeps = [&](int col0, int ncols, hipStream_t st) -> hipError_t {
    // forward sweep: Y_r -= Lh_rI Y_I (r > I) and dW_I = P_I Y_I. After the first
    // block the blocks go in pairs (I, I+1): one launch finishes Y_{I+1} and forms
    // dW_I, the next updates every later block with both (depth 512, so the
    // read-modify-write of the right-hand side below is shared by two blocks)
    // and forms dW_{I+1}. The A operand is the mirrored Lh above the diagonal,
    // whose rows I*256 .. of blocks I and I+1 are consecutive. Row pointers of
    // the right-hand side, Y and dW are taken at column 0 and moved to col0 here.
    auto fwd_launch = [&](const float* A, float* Ydst, const float* Ysrc, int M, const float* Bsum, int Ksum,
                          int P, const float* Bp, int Kp) -> hipError_t {
      GemmArgs g = {};
      int j = 0;
      if (M > 0) {
        g.job[j] = GemmJob{A, Ydst + col0, M, d, d_out, 1, Ysrc + col0};
        g.job[j].la = g.job[j].lc = ws;
        g.job[j].B = Bsum + col0;
        g.job[j].K = Ksum;
        ++j;
      }
      g.job[j] = GemmJob{pinv + (int64_t)P * kBb * kBb, delta_w + (int64_t)P * kBb * d_out + col0, Kp, kBb, d_out, 0};
      g.job[j].la = ws;
      g.job[j].lc = dws;
      g.job[j].B = Bp + col0;
      g.job[j].K = Kp;
      ++j;
      g.n_jobs = j;
      g.lb = ws;
      g.B = Bp + col0;
      g.N = ncols;
      g.K = Kp;
      g.ldb = d_out;
      return launch_gemm(g, nl, st);
    };
    hipError_t e;
    // the first step reads the right-hand side C itself (Y = C before any update)
    e = fwd_launch(lup(0, 1), yblk(Y, 1), yblk(C, 1), d - kBb, C, kblk(0), 0, C, kblk(0));
    if (e != hipSuccess) return e;
    for (int I = 1; I < nb; I += 2) {
      if (I + 1 == nb) {
        e = fwd_launch(nullptr, Y, Y, 0, Y, 0, I, yblk(Y, I), kblk(I));
        if (e != hipSuccess) return e;
        break;
      }
      e = fwd_launch(lup(I, I + 1), yblk(Y, I + 1), yblk(Y, I + 1), kblk(I + 1), yblk(Y, I), kBb, I, yblk(Y, I),
                     kBb);
      if (e != hipSuccess) return e;
      const int below = d - (I + 2) * kBb;
      e = fwd_launch(below > 0 ? lup(I, I + 2) : nullptr, below > 0 ? yblk(Y, I + 2) : Y,
                     below > 0 ? yblk(Y, I + 2) : Y, max(below, 0), yblk(Y, I), kBb + kblk(I + 1), I + 1,
                     yblk(Y, I + 1), kblk(I + 1));
      if (e != hipSuccess) return e;
    }
    // backward sweep: dW_I -= Lh_JI^T dW_J (I < J), from the last block down in
    // pairs (J, J-1): one launch finishes dW_{J-1}, the next updates every earlier
    // block with both (rows (J-1)*256 .. of L, depth 512); rows from row0 on
    auto bwd_launch = [&](int J, int M, int K, int row0) -> hipError_t {
      GemmArgs g = {};
      g.job[0] = GemmJob{L + (int64_t)J * kBb * d + row0, delta_w + (int64_t)row0 * d_out + col0, M, d, d_out, 1};
      g.job[0].la = ws;
      g.job[0].lc = dws;
      g.lb = dws;
      g.n_jobs = 1;
      g.B = yblk(delta_w, J) + col0;
      g.N = ncols;
      g.K = K;
      g.ldb = d_out;
      return launch_gemm(g, nl, st);
    };
    for (int J = nb - 1; J >= 1; J -= 2) {
      e = bwd_launch(J, kBb, kblk(J), (J - 1) * kBb);
      if (e != hipSuccess) return e;
      if (J - 1 >= 1) {
        e = bwd_launch(J - 1, (J - 1) * kBb, kBb + kblk(J), 0);
        if (e != hipSuccess) return e;
      }
    }
    return hipSuccess;
  };
  {
    SideStream* side = d_out >= 2 * kSweepCols ? side_stream(d) : nullptr;
    hipError_t e;
    if (side != nullptr) {
      std::lock_guard<std::mutex> lock(g_side_mu);
      const int half = (d_out / 2 + kSweepCols - 1) / kSweepCols * kSweepCols;
      if ((e = hipEventRecord(side->fork, stream)) != hipSuccess) return e;
      if ((e = hipStreamWaitEvent(side->s, side->fork, 0)) != hipSuccess) return e;
      if ((e = sweeps(0, half, stream)) != hipSuccess) return e;
      if ((e = sweeps(half, d_out - half, side->s)) != hipSuccess) return e;
      if ((e = hipEventRecord(side->join, side->s)) != hipSuccess) return e;
      if ((e = hipStreamWaitEvent(stream, side->join, 0)) != hipSuccess) return e;
    } else if ((e = sweeps(0, d_out, stream)) != hipSuccess) {
      return e;
    }
  }
  // the P_I area is free once the forward sweep has run: it holds the partial sums
  const int64_t n = (int64_t)d * d_out;
  hipLaunchKernelGGL(eps_partial_kernel, dim3(kEpsBlocks, nl), dim3(kThreads), 0, stream, delta_w, C, n,
                     (double*)pinv, ws, dws);
  hipLaunchKernelGGL(eps_final_kernel, dim3(1, nl), dim3(kThreads), 0, stream, (const double*)pinv, kEpsBlocks,
                     w.scalars, (double)lambda, (const int*)w.status, w.eps_out, w.status_out, ws);
  return hipGetLastError();
}

}  // namespace ispa
