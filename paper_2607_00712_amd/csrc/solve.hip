// Closed-form modulation dW = (G + lambda I)^-1 C for gfx950 (CDNA4).
//
// Operation (arXiv 2607.00712, Sec. 3.2, Eq. 5): one D x D SPD system with
// D_out right-hand sides, solved at the end of warmup. The "inversion" is
// carried out as a Cholesky factorisation A = L L^T of A = G + lambda I and two
// triangular solves L Z = C, L^T dW = Z, all in fp32. Eq. 6's feasibility score
// follows from the same quantities: eps = s - <dW, C> - lambda ||dW||^2.
//
// Factorisation: blocked right-looking Cholesky with panel width kNb = 64.
//   panel step k:  every workgroup loads the (already updated) diagonal block
//                  into LDS and factors it (unblocked, column by column);
//                  workgroup 0 writes L_kk and raises the status flag on a
//                  non-positive pivot; the other workgroups each solve one
//                  64-row block below it, L_ik = A_ik L_kk^-T.
//   update step k: A22 -= L21 L21^T on the lower triangle of 64x64 tiles,
//                  fp32 FMA with a 4x4 register micro-tile per thread.
// Triangular solves: left-looking by 64-row block rows; one launch per block
// row and direction, parallel over 64-column tiles of the right-hand side:
//   forward  Z_i  = L_ii^-1 (C_i - sum_{j<i} L_ij Z_j)
//   backward dW_i = L_ii^-T (Z_i - sum_{j>i} L_ji^T dW_j)
// The GEMM part of each launch runs over 64-deep slabs staged in LDS; the
// diagonal solve runs in LDS with one column per thread.
#include "ispa_internal.h"

#include <math.h>

namespace ispa {
namespace {

constexpr int kNb = 64;
constexpr int kThreads = 256;
constexpr int kPad = 65;  // LDS row stride (floats) for 64-wide blocks

// L = lower(G) + lambda I, zero above the diagonal. n x n, row-major.
__global__ void chol_init_kernel(const float* G, float* L, int n, float lambda, int* status) {
  const int64_t total = (int64_t)n * n;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int r = (int)(i / n), c = (int)(i % n);
    float v = 0.f;
    if (c < r) v = G[i];
    else if (c == r) v = G[i] + lambda;
    L[i] = v;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) *status = 0;
}

// Unblocked Cholesky of the nb x nb block in LDS (lower), all threads.
__device__ void factor_diag(float (*a)[kPad], int nb, int* bad) {
  for (int j = 0; j < nb; ++j) {
    __syncthreads();
    if (threadIdx.x == 0) {
      float d = a[j][j];
      if (!(d > 0.f)) { *bad = 1; d = 1.f; }
      a[j][j] = sqrtf(d);
    }
    __syncthreads();
    const float inv = 1.f / a[j][j];
    for (int i = j + 1 + (int)threadIdx.x; i < nb; i += blockDim.x) a[i][j] *= inv;
    __syncthreads();
    // trailing update of the block's lower triangle
    const int m = nb - j - 1;
    for (int t = threadIdx.x; t < m * m; t += blockDim.x) {
      const int i = j + 1 + t / m, c = j + 1 + t % m;
      if (c <= i) a[i][c] -= a[i][j] * a[c][j];
    }
  }
  __syncthreads();
}

// Panel step at column k: blockIdx.x == 0 writes the diagonal block; block b > 0
// solves rows [k + b*nb, k + (b+1)*nb) of the panel.
__global__ __launch_bounds__(kThreads) void chol_panel_kernel(float* L, int n, int k, int* status) {
  __shared__ float dg[kNb][kPad];
  __shared__ float rw[kNb][kPad];
  __shared__ int bad;
  const int nb = min(kNb, n - k);
  if (threadIdx.x == 0) bad = 0;
  for (int t = threadIdx.x; t < nb * nb; t += blockDim.x) {
    const int i = t / nb, c = t % nb;
    dg[i][c] = c <= i ? L[(int64_t)(k + i) * n + k + c] : 0.f;
  }
  factor_diag(dg, nb, &bad);
  if (blockIdx.x == 0) {
    for (int t = threadIdx.x; t < nb * nb; t += blockDim.x) {
      const int i = t / nb, c = t % nb;
      if (c <= i) L[(int64_t)(k + i) * n + k + c] = dg[i][c];
    }
    if (threadIdx.x == 0 && bad) atomicOr(status, 1);
    return;
  }
  const int r0 = k + nb + (blockIdx.x - 1) * kNb;
  if (r0 >= n) return;
  const int rows = min(kNb, n - r0);
  for (int t = threadIdx.x; t < rows * nb; t += blockDim.x) {
    const int i = t / nb, c = t % nb;
    rw[i][c] = L[(int64_t)(r0 + i) * n + k + c];
  }
  __syncthreads();
  // X L^T = B row by row: x_c = (b_c - sum_{j<c} x_j L_cj) / L_cc
  if ((int)threadIdx.x < rows) {
    const int i = threadIdx.x;
    for (int c = 0; c < nb; ++c) {
      float v = rw[i][c];
      for (int j = 0; j < c; ++j) v -= rw[i][j] * dg[c][j];
      rw[i][c] = v / dg[c][c];
    }
  }
  __syncthreads();
  for (int t = threadIdx.x; t < rows * nb; t += blockDim.x) {
    const int i = t / nb, c = t % nb;
    L[(int64_t)(r0 + i) * n + k + c] = rw[i][c];
  }
}

// Trailing update A22 -= P P^T for the lower triangle, P = L[k+nb:, k:k+nb].
__global__ __launch_bounds__(kThreads) void chol_update_kernel(float* L, int n, int k) {
  __shared__ float pa[kNb][kPad];
  __shared__ float pb[kNb][kPad];
  const int nb = min(kNb, n - k);
  const int base = k + nb;
  // lower-triangle tile index -> (ti, tj)
  const int t = blockIdx.x;
  int ti = (int)((sqrtf(8.f * t + 1.f) - 1.f) * 0.5f);
  while ((ti + 1) * (ti + 2) / 2 <= t) ++ti;
  while (ti * (ti + 1) / 2 > t) --ti;
  const int tj = t - ti * (ti + 1) / 2;
  const int r0 = base + ti * kNb, c0 = base + tj * kNb;
  if (r0 >= n || c0 >= n) return;
  for (int e = threadIdx.x; e < kNb * nb; e += blockDim.x) {
    const int i = e / nb, c = e % nb;
    pa[i][c] = r0 + i < n ? L[(int64_t)(r0 + i) * n + k + c] : 0.f;
    pb[i][c] = c0 + i < n ? L[(int64_t)(c0 + i) * n + k + c] : 0.f;
  }
  __syncthreads();
  const int tr = (threadIdx.x / 16) * 4, tc = (threadIdx.x % 16) * 4;
  float acc[4][4] = {};
  for (int c = 0; c < nb; ++c) {
    float a[4], b[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) { a[u] = pa[tr + u][c]; b[u] = pb[tc + u][c]; }
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int v = 0; v < 4; ++v) acc[u][v] = fmaf(a[u], b[v], acc[u][v]);
  }
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int r = r0 + tr + u, c = c0 + tc + v;
      if (r < n && c <= r) L[(int64_t)r * n + c] -= acc[u][v];
    }
}

// Forward (dir = 0) or backward (dir = 1) solve of block row bi for a 64-column
// tile of the right-hand side. rhs is C (forward) or Z (backward); X holds Z
// (forward output, in place for backward).
__global__ __launch_bounds__(kThreads) void trsm_kernel(const float* L, const float* rhs, float* X,
                                                       int n, int n_out, int bi, int dir) {
  __shared__ float lt[kNb][kPad];   // L slab (64 x 64)
  __shared__ float xt[kNb][kPad];   // X slab (64 rows x 64 cols)
  __shared__ float acc_s[kNb][kPad];
  const int r0 = bi * kNb;
  const int nb = min(kNb, n - r0);
  const int c0 = blockIdx.x * kNb;
  const int tr = (threadIdx.x / 16) * 4, tc = (threadIdx.x % 16) * 4;
  float acc[4][4] = {};
  const int nblk = (n + kNb - 1) / kNb;
  // GEMM over the already-solved block rows
  const int jb0 = dir == 0 ? 0 : bi + 1;
  const int jb1 = dir == 0 ? bi : nblk;
  for (int jb = jb0; jb < jb1; ++jb) {
    const int j0 = jb * kNb;
    const int kb = min(kNb, n - j0);
    __syncthreads();
    for (int e = threadIdx.x; e < kNb * kNb; e += blockDim.x) {
      const int i = e / kNb, c = e % kNb;
      // forward: lt[i][c] = L[r0+i][j0+c]; backward: lt[i][c] = L[j0+c][r0+i] (= L^T)
      float lv = 0.f;
      if (i < nb && c < kb) lv = dir == 0 ? L[(int64_t)(r0 + i) * n + j0 + c] : L[(int64_t)(j0 + c) * n + r0 + i];
      lt[i][c] = lv;
      float xv = 0.f;
      if (i < kb && c0 + c < n_out) xv = X[(int64_t)(j0 + i) * n_out + c0 + c];
      xt[i][c] = xv;
    }
    __syncthreads();
    for (int c = 0; c < kNb; ++c) {
      float a[4], b[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) { a[u] = lt[tr + u][c]; b[u] = xt[c][tc + u]; }
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int v = 0; v < 4; ++v) acc[u][v] = fmaf(a[u], b[v], acc[u][v]);
    }
  }
  __syncthreads();
  // right-hand side minus the GEMM part, and the diagonal block
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int r = tr + u, c = tc + v;
      float b = 0.f;
      if (r < nb && c0 + c < n_out) b = rhs[(int64_t)(r0 + r) * n_out + c0 + c];
      acc_s[r][c] = b - acc[u][v];
    }
  for (int e = threadIdx.x; e < kNb * kNb; e += blockDim.x) {
    const int i = e / kNb, c = e % kNb;
    lt[i][c] = (i < nb && c < nb) ? L[(int64_t)(r0 + i) * n + r0 + c] : (i == c ? 1.f : 0.f);
  }
  __syncthreads();
  if ((int)threadIdx.x < kNb) {
    const int c = threadIdx.x;
    if (dir == 0) {
      for (int i = 0; i < nb; ++i) {
        float v = acc_s[i][c];
        for (int j = 0; j < i; ++j) v -= lt[i][j] * acc_s[j][c];
        acc_s[i][c] = v / lt[i][i];
      }
    } else {
      for (int i = nb - 1; i >= 0; --i) {
        float v = acc_s[i][c];
        for (int j = i + 1; j < nb; ++j) v -= lt[j][i] * acc_s[j][c];
        acc_s[i][c] = v / lt[i][i];
      }
    }
  }
  __syncthreads();
  for (int e = threadIdx.x; e < kNb * kNb; e += blockDim.x) {
    const int i = e / kNb, c = e % kNb;
    if (i < nb && c0 + c < n_out) X[(int64_t)(r0 + i) * n_out + c0 + c] = acc_s[i][c];
  }
}

// scalars[0] += <dW, C>, scalars[1] += ||dW||^2
__global__ __launch_bounds__(kThreads) void eps_kernel(const float* dw, const float* C, int64_t n,
                                                      double* scalars) {
  __shared__ double red[2][kThreads / 64];
  double a = 0, b = 0;
  for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n; i += (int64_t)gridDim.x * kThreads) {
    const double w = dw[i];
    a += w * (double)C[i];
    b += w * w;
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) { a += __shfl_xor(a, o); b += __shfl_xor(b, o); }
  if ((threadIdx.x & 63) == 0) { red[0][threadIdx.x >> 6] = a; red[1][threadIdx.x >> 6] = b; }
  __syncthreads();
  if (threadIdx.x == 0) {
    double ta = 0, tb = 0;
    for (int w = 0; w < kThreads / 64; ++w) { ta += red[0][w]; tb += red[1][w]; }
    atomicAdd(&scalars[0], ta);
    atomicAdd(&scalars[1], tb);
  }
}

__global__ void zero_scalars_kernel(double* s) {
  if (threadIdx.x < 2) s[threadIdx.x] = 0.0;
}

}  // namespace

hipError_t launch_solve(const float* G, const float* C, int d, int d_out, float lambda,
                        float* delta_w, const SolveWork& w, hipStream_t stream) {
  const int64_t dd = (int64_t)d * d;
  int grid = (int)((dd + 255) / 256);
  if (grid > 4096) grid = 4096;
  hipLaunchKernelGGL(chol_init_kernel, dim3(grid), dim3(256), 0, stream, G, w.L, d, lambda, w.status);
  const int nblk = (d + kNb - 1) / kNb;
  for (int kb = 0; kb < nblk; ++kb) {
    const int k = kb * kNb;
    const int below = nblk - kb - 1;
    hipLaunchKernelGGL(chol_panel_kernel, dim3(1 + below), dim3(kThreads), 0, stream, w.L, d, k, w.status);
    if (below > 0) {
      hipLaunchKernelGGL(chol_update_kernel, dim3(below * (below + 1) / 2), dim3(kThreads), 0, stream,
                         w.L, d, k);
    }
  }
  const int col_tiles = (d_out + kNb - 1) / kNb;
  for (int bi = 0; bi < nblk; ++bi)
    hipLaunchKernelGGL(trsm_kernel, dim3(col_tiles), dim3(kThreads), 0, stream, w.L, C, delta_w, d, d_out,
                       bi, 0);
  for (int bi = nblk - 1; bi >= 0; --bi)
    hipLaunchKernelGGL(trsm_kernel, dim3(col_tiles), dim3(kThreads), 0, stream, w.L, delta_w, delta_w, d,
                       d_out, bi, 1);
  hipLaunchKernelGGL(zero_scalars_kernel, dim3(1), dim3(64), 0, stream, w.scalars);
  const int64_t n = (int64_t)d * d_out;
  int eg = (int)((n + kThreads - 1) / kThreads);
  if (eg > 1024) eg = 1024;
  hipLaunchKernelGGL(eps_kernel, dim3(eg), dim3(kThreads), 0, stream, delta_w, C, n, w.scalars);
  return hipGetLastError();
}

}  // namespace ispa
