// Shared definitions of the two expert-FFN GEMM kernels.
#pragma once

#include "common.h"
#include "kernels.h"

namespace moe {

// out[row][n] = epilogue( sum_c x[row][c] * W(g, n, c) ) for every row of
// group g, with W(g, n, c) = w[g*group_stride + col_offset(c) + n*ldw] and
// col_offset(c) = c for a single K segment (kseg >= K) or
// (c / kseg)*seg_stride + c % kseg for K stacked over several experts.
// GATED kernels read two such matrices (w0 = gate, w1 = up) and write
// silu(gate) * up.  x rows have stride K and out rows stride N; row r of the
// grouped activation matrix is x[x_rows[r]] when x_rows != nullptr.
//
// Chunk-blocked layout (weight-streaming kernel with device offsets only, K
// and N multiples of 16): a group's rows are cut into chunks of 32, the last
// one padded (with zeros, since padded inputs give zero outputs), chunk j of
// group g being global chunk sum_{g' < g} ceil(rows_g' / 32) + j.  Chunk c of
// a matrix with C columns holds C/16 blocks of 1 KB, block s holding column
// 16s + 8h + e of chunk row t at element 8*(32*h + t) + e: exactly the B
// operand of one v_mfma_f32_32x32x16_bf16 (lane 32h + t, 8 values), so a
// wave loads it as one contiguous 1 KB.  x_blocked reads x in this layout;
// out_blocked writes out in it, padding rows included.
struct GemmArgs {
  const uint16_t* x;
  const int32_t* x_rows;
  int x_row_count;  // rows of x when x_rows is set
  bool x_blocked, out_blocked;
  const int32_t* offsets;  // [groups+1] device, or nullptr for one group of static_rows
  int static_rows;
  int groups;
  const uint16_t* w0;
  const uint16_t* w1;
  uint16_t* out;
  int K, N, kseg, ldw;
  size_t seg_stride, group_stride;
};

__device__ __forceinline__ size_t weight_col_offset(const GemmArgs& a, int c) {
  if (a.kseg >= a.K) return static_cast<size_t>(c);
  const int q = c / a.kseg;
  return static_cast<size_t>(q) * a.seg_stride + static_cast<size_t>(c - q * a.kseg);
}

hipError_t launch_skinny(const Segments& seg, const GemmArgs& a, bool gated, hipStream_t st);
// Host-side size limits of the weight-streaming kernel (launch_skinny
// refuses arguments that fail this check; it also requires device offsets
// for the blocked layouts).
bool skinny_ok(const GemmArgs& a);
constexpr int kChunkRows = kChunkRowsHost;
constexpr int kBlockElems = 512;  // one 1 KB block of the chunk-blocked layout
hipError_t launch_tiled(const Segments& seg, const GemmArgs& a, bool gated, hipStream_t st);

// Largest per-group row count routed to the weight-streaming kernel.
constexpr int kSkinnyMaxRows = 64;

}  // namespace moe
