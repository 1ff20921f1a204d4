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
// grouped activation matrix is x[x_rows[r]] when x_rows != nullptr
// (weight-streaming kernel only).
struct GemmArgs {
  const uint16_t* x;
  const int32_t* x_rows;
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
hipError_t launch_tiled(const Segments& seg, const GemmArgs& a, bool gated, hipStream_t st);

// Largest per-group row count routed to the weight-streaming kernel.
constexpr int kSkinnyMaxRows = 64;

}  // namespace moe
