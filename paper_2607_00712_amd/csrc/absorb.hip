// Layer absorption after warmup for gfx950 (CDNA4): the in-place weight
// update of an L-Layer and its KV cache after the permanent eviction.
//
// Operation (arXiv 2607.00712, Sec. 3.3): each selected layer takes
// W_new = W + dW for its output projection, and drops its history so that it
// keeps only the local context of Sec. 3.4, Eq. 7 (the sink prefix and the
// most recent keys). Both are one-off, bandwidth-bound copies; they are kernels
// so that no step of the path runs on the host.
//
// Weight update: W stored [d_in, d_out] (the row-vector form of Eq. 4) adds dW
// element-wise; stored [d_out, d_in] (a linear layer's weight) it adds dW^T,
// staged through LDS in 32 x 32 tiles so that both sides are read and written
// in rows. bf16 weights take the fp32 sum rounded to nearest even.
// KV ring: an L-Layer's cache is [sink rows | window rows]; the window rows form
// a ring in which key number h (counting window keys since the eviction) lives
// at row sink + h mod window. Attention does not depend on the order of its
// keys, so the ring is attended as one contiguous range of rows.
#include "ispa_internal.h"

namespace ispa {
namespace {

constexpr int kTile = 32;

__device__ __forceinline__ float load_w(const float* p) { return *p; }
__device__ __forceinline__ float load_w(const __bf16* p) { return (float)*p; }
__device__ __forceinline__ void store_w(float* p, float x) { *p = x; }
__device__ __forceinline__ void store_w(__bf16* p, float x) { *p = (__bf16)x; }

// W[i][j] += dW[i][j], W and dW [d_in, d_out]
template <typename T>
__global__ void inject_kernel(T* W, const float* dW, int64_t n) {
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += (int64_t)gridDim.x * blockDim.x)
    store_w(W + e, load_w(W + e) + dW[e]);
}

// W[j][i] += dW[i][j], W [d_out, d_in], dW [d_in, d_out]; block (32, 8) per
// 32 x 32 tile of W
template <typename T>
__global__ void inject_t_kernel(T* W, const float* dW, int d_in, int d_out) {
  __shared__ float t[kTile][kTile + 1];
  const int j0 = blockIdx.y * kTile;  // rows of W = columns of dW
  const int i0 = blockIdx.x * kTile;  // columns of W = rows of dW
  // read the dW tile [i0.., j0..] in rows of dW
  for (int r = threadIdx.y; r < kTile; r += blockDim.y) {
    const int i = i0 + r, j = j0 + threadIdx.x;
    t[r][threadIdx.x] = (i < d_in && j < d_out) ? dW[(int64_t)i * d_out + j] : 0.f;
  }
  __syncthreads();
  // update the W tile [j0.., i0..] in rows of W
  for (int r = threadIdx.y; r < kTile; r += blockDim.y) {
    const int j = j0 + r, i = i0 + threadIdx.x;
    if (j < d_out && i < d_in) {
      T* p = W + (int64_t)j * d_in + i;
      store_w(p, load_w(p) + t[threadIdx.x][r]);
    }
  }
}

// Row copies of K and V: segment s moves rows [src, src + n) of the source to
// rows [dst, dst + n) of the destination; rows are `row16` 16-byte chunks.
struct RowCopies {
  int64_t src[3], dst[3], n[3];
  int n_seg;
};

__global__ void kv_copy_kernel(const uint4* k_src, const uint4* v_src, uint4* k_dst, uint4* v_dst, int64_t row16,
                               RowCopies c) {
  int64_t total = 0;
  for (int s = 0; s < c.n_seg; ++s) total += c.n[s];
  const int64_t chunks = total * row16;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < chunks; e += (int64_t)gridDim.x * blockDim.x) {
    int64_t row = e / row16;
    const int64_t col = e - row * row16;
    int s = 0;
    while (row >= c.n[s]) {
      row -= c.n[s];
      ++s;
    }
    const int64_t so = (c.src[s] + row) * row16 + col, d = (c.dst[s] + row) * row16 + col;
    k_dst[d] = k_src[so];
    v_dst[d] = v_src[so];
  }
}

}  // namespace

hipError_t launch_inject(void* W, int dtype, bool transposed, const float* dW, int d_in, int d_out,
                         hipStream_t stream) {
  if (!transposed) {
    const int64_t n = (int64_t)d_in * d_out;
    const int blocks = (int)((n + 255) / 256 < 8192 ? (n + 255) / 256 : 8192);
    if (dtype == 0)
      hipLaunchKernelGGL(inject_kernel<__bf16>, dim3(blocks), dim3(256), 0, stream, (__bf16*)W, dW, n);
    else
      hipLaunchKernelGGL(inject_kernel<float>, dim3(blocks), dim3(256), 0, stream, (float*)W, dW, n);
  } else {
    const dim3 grid((d_in + kTile - 1) / kTile, (d_out + kTile - 1) / kTile);
    if (dtype == 0)
      hipLaunchKernelGGL(inject_t_kernel<__bf16>, grid, dim3(kTile, 8), 0, stream, (__bf16*)W, dW, d_in, d_out);
    else
      hipLaunchKernelGGL(inject_t_kernel<float>, grid, dim3(kTile, 8), 0, stream, (float*)W, dW, d_in, d_out);
  }
  return hipGetLastError();
}

hipError_t launch_kv_copy(const void* k_src, const void* v_src, void* k_dst, void* v_dst, int64_t row_bytes,
                          const int64_t* src, const int64_t* dst, const int64_t* n, int n_seg, hipStream_t stream) {
  RowCopies c;
  int64_t total = 0;
  for (int s = 0; s < 3; ++s) {
    c.src[s] = s < n_seg ? src[s] : 0;
    c.dst[s] = s < n_seg ? dst[s] : 0;
    c.n[s] = s < n_seg ? n[s] : 0;
    total += c.n[s];
  }
  c.n_seg = n_seg;
  if (total == 0) return hipSuccess;
  const int64_t row16 = row_bytes / 16;
  const int64_t chunks = total * row16;
  const int blocks = (int)((chunks + 255) / 256 < 8192 ? (chunks + 255) / 256 : 8192);
  hipLaunchKernelGGL(kv_copy_kernel, dim3(blocks), dim3(256), 0, stream, (const uint4*)k_src, (const uint4*)v_src,
                     (uint4*)k_dst, (uint4*)v_dst, row16, c);
  return hipGetLastError();
}

}  // namespace ispa
