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

// Split of the work over workgroups (used when whole work items would leave
// part of the chip idle). The units are (work item, key tile) pairs in
// item-major order, U = work items x tiles per item; segment g of G covers
// units [g U / G, (g + 1) U / G). A piece is the part of one work item inside
// one segment; a piece that does not cover all tiles of its item (or all its
// local tiles) leaves its normalised output and LSE in a partial slot for
// attn_merge_split.
struct AttnSplit {
  int64_t units;       // U
  int32_t n_seg;       // G; 0: one whole work item per workgroup, no partials
  int32_t max_pieces;  // partial slots per segment
  float* part_o;       // [G * max_pieces][2][kAttnBq][head_dim]: [.][0] end state, [.][1] local set
  float* part_lse;     // [G * max_pieces][2][kAttnBq]
  // counters [work item][2 streams][4 waves] of the split fold (the assembly
  // kernel's pieces complete their work items themselves); null: the merge
  // kernel completes them after the launch
  uint32_t* ctr;
  size_t lse_offset, ctr_offset;  // byte offsets of part_lse and ctr in the workspace
};
constexpr int kAttnBq = 256;  // queries per work item

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
  AttnSplit split;
};

// Tiles of 64 keys visited for each work item, and those of the local set.
int attn_tiles(const AttnRanges& r, int* n_tiles_local);
// Compute units of the current device.
int attn_cu_count();
// Split plan for a launch: segments < 0 never splits, 0 splits when whole work
// items would fill the chip poorly, > 0 forces that many segments. Fills
// units/n_seg/max_pieces (n_seg = 0: no split) and returns the workspace bytes.
size_t attn_plan_split(const AttnArgs& a, int head_dim, int segments, AttnSplit* s);
hipError_t launch_attn_chunk(const AttnArgs& a, int head_dim, hipStream_t stream);
// The hand-scheduled head_dim-128 kernel (attn_fast.cpp): whether it takes
// this launch (its 32-bit work arithmetic fits and its code object loaded on
// the current device), and the launch itself (the split's merge excluded).
bool attn_fast_eligible(const AttnArgs& a, int head_dim);
hipError_t launch_attn_fast(const AttnArgs& a, hipStream_t stream);
// out = 0, lse = -inf (attention over an empty key set)
hipError_t launch_attn_empty(float* out, float* lse, int64_t n_q, int64_t n_heads, int head_dim,
                             hipStream_t stream);
// Eq. 11-12 merge of two results over disjoint key sets (out may alias a or b).
hipError_t launch_attn_merge2(const float* o_a, const float* lse_a, const float* o_b, const float* lse_b,
                              int64_t n_q, int64_t n_heads, int head_dim, float* out, float* lse,
                              hipStream_t stream);

// ---- statistics (stats.hip) ----
// The discrepancy kernel leaves one fp64 norm partial per workgroup in
// sq_part (discrepancy_grid of them, at most kDiscMaxGrid); the Gram launch
// that follows on the stream adds them to *sq_norm in workgroup order.
constexpr int kDiscMaxGrid = 512;
int discrepancy_grid(int64_t rows, int d_in, int d_out);
hipError_t launch_discrepancy(const void* x, int x_dtype, const void* y_full, const void* y_local,
                              int y_dtype, int64_t rows, int d_in, int d_out,
                              uint16_t* x_bf16, uint16_t* r_bf16, double* sq_part, hipStream_t stream);
// Gram tiles of (d_in, d_out); below kGramSplitTiles the rows are split in two
// inside each workgroup.
constexpr int kGramSplitTiles = 256;
int gram_tiles(int d_in, int d_out);
hipError_t launch_gram(const uint16_t* x, const uint16_t* r, int64_t rows, int d_in, int d_out,
                       float* G, float* C, const double* sq_part, int n_sq_part, double* sq_norm,
                       float* scratch, size_t scratch_bytes, hipStream_t stream);
hipError_t launch_zero(void* p, size_t bytes, hipStream_t stream);
// the hand-scheduled Gram kernel (gram_fast.cpp): widths that are multiples of
// 256; tiles computed whole (n_whole) or as 2^log_pieces row pieces of `split`
// stages (n_split tiles), the later pieces' sums in (2^log_pieces - 1) x n_split
// scratch slots of 256 x 256 fp32 that gram_fixup adds after the launch
struct GramFastPlan {
  int log_pieces, n_whole, n_split, split;
};
bool gram_fast_plan(int64_t rows, int d_in, int d_out, size_t scratch_bytes, GramFastPlan* plan);
// scratch that gram_fast_plan may ask for at these widths on this device
size_t gram_fast_scratch_bytes(int d_in, int d_out);
hipError_t launch_gram_fast(const uint16_t* x, const uint16_t* r, int64_t rows, int d_in, int d_out, float* G,
                            float* C, float* scratch, const GramFastPlan& plan, hipStream_t stream);

// ---- absorption (absorb.hip) ----
// W += dW (transposed: W[j][i] += dW[i][j]); dtype 0 bf16, 1 fp32
hipError_t launch_inject(void* W, int dtype, bool transposed, const float* dW, int d_in, int d_out,
                         hipStream_t stream);
// up to 3 row copies of K and V (rows of row_bytes, a multiple of 16)
hipError_t launch_kv_copy(const void* k_src, const void* v_src, void* k_dst, void* v_dst, int64_t row_bytes,
                          const int64_t* src, const int64_t* dst, const int64_t* n, int n_seg, hipStream_t stream);

// ---- projection (project.hip) ----
// y = a w^T: a bf16 [n, d_in], w bf16 [d_out, d_in], y fp32 or bf16 [n, d_out];
// d_in a multiple of 32
hipError_t launch_project(const void* a, const void* w, int64_t n, int d_in, int d_out, void* y, int y_bf16,
                          int n_cu, hipStream_t stream);
// W8A8: y = (qa qw^T) * sa[row] * sw[col]; qa int8 [n, d_in], qw int8
// [d_out, d_in]; d_in a multiple of 64
hipError_t launch_project_w8a8(const int8_t* qa, const float* sa, const int8_t* qw, const float* sw, int64_t n,
                               int d_in, int d_out, void* y, int y_bf16, int n_cu, hipStream_t stream);
// the hand-scheduled projection kernels (proj_fast.cpp): d_out a multiple of
// 256 and at least 512 rows; with i8 the W8A8 form (sa, sw its scales)
bool proj_fast_eligible(int64_t n, int d_in, int d_out, bool i8);
hipError_t launch_proj_fast(const void* a, const void* w, const float* sa, const float* sw, int64_t n, int d_in,
                            int d_out, void* y, int y_bf16, bool i8, int n_cu, hipStream_t stream);
// per-row int8 codes and scales of x (fp32 or bf16) [rows, cols]; cols a
// multiple of 8, x 16-byte aligned
hipError_t launch_quantize_rows(const void* x, int x_bf16, int64_t rows, int cols, int8_t* q, float* scale,
                                hipStream_t stream);

// ---- solve (solve.hip) ----
struct SolveWork {
  float* L;          // [d, d] factor (lower triangle)
  float* work;       // [d, d_out] right-hand side being reduced
  float* dinv;       // [ceil(d/64), 64, 64] inverses of the diagonal blocks of L
  int* status;       // device int: 0 ok, 1 not SPD
  double* scalars;   // device: [0] s (input), then [2] <dW, C>, [3] ||dW||^2, [4] eps, [5] status
  double* eps_out = nullptr;  // optional device copies of eps and the status word ([n_layers] each)
  int* status_out = nullptr;
  // batched solves: n_layers systems whose workspaces (every pointer above
  // except the outputs) are ws_stride bytes apart and whose dW are dw_stride
  // bytes apart
  int n_layers = 1;
  int64_t ws_stride = 0;
  int64_t dw_stride = 0;
};
size_t solve_dinv_bytes(int d);
// host-only check of a single layer's look-ahead factorisation schedule (0: valid)
int solve_lookahead_check(int nblk, int n_cu);
hipError_t launch_solve(const float* G, const float* C, int d, int d_out, float lambda,
                        float* delta_w, const SolveWork& w, hipStream_t stream);

}  // namespace ispa
