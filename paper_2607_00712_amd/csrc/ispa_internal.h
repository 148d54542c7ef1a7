// Internal declarations shared by the host layer and the kernel files of
// libispa (gfx950 only). Nothing here is part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

#include "ispa.h"

namespace ispa {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

#define ISPA_LDS __attribute__((address_space(3)))

// Key ranges visited by one attention launch. Ranges [0, n_local) form the
// local set (sink prefix, then window tail); range n_local, if present, is the
// history. Each range is a contiguous run of cache rows.
struct AttnRanges {
  int64_t begin[3];
  int64_t end[3];
  int n_local;   // 1 or 2
  int n_total;   // n_local or n_local + 1
};

struct AttnArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  float* out;
  float* lse;
  float* out_local;   // non-null: dual-stream launch
  float* lse_local;
  int64_t ld;         // row stride of q/k/v/out in elements (n_heads * head_dim)
  int32_t n_q;
  int32_t n_heads;
  float scale_log2;   // logit scale * log2(e)
  float scale;        // logit scale (for the natural-log LSE)
  AttnRanges r;
};

hipError_t launch_attn_chunk(const AttnArgs& a, int head_dim, hipStream_t stream);

// ---- statistics (stats.hip) ----
hipError_t launch_discrepancy(const void* x, int x_dtype, const void* y_full, const void* y_local,
                              int y_dtype, int64_t rows, int d_in, int d_out,
                              uint16_t* x_bf16, uint16_t* r_bf16, double* sq_norm,
                              hipStream_t stream);
hipError_t launch_gram(const uint16_t* x, const uint16_t* r, int64_t rows, int d_in, int d_out,
                       float* G, float* C, hipStream_t stream);
hipError_t launch_zero(void* p, size_t bytes, hipStream_t stream);

// ---- solve (solve.hip) ----
struct SolveWork {
  float* L;          // [d, d] factor (lower triangle)
  float* work;       // [d, d_out] right-hand side being reduced
  float* dinv;       // [ceil(d/64), 64, 64] inverses of the diagonal blocks of L
  int* status;       // device int: 0 ok, 1 not SPD
  double* scalars;   // device: [0] <dW, C>, [1] ||dW||^2
};
size_t solve_dinv_bytes(int d);
hipError_t launch_solve(const float* G, const float* C, int d, int d_out, float lambda,
                        float* delta_w, const SolveWork& w, hipStream_t stream);

}  // namespace ispa
