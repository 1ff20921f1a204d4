// Expert FFN for decode-sized batches: weight streaming.
//
// With at most a few dozen rows per expert the grouped GEMM is bound by
// reading the experts' weights from HBM once.  The weights therefore take
// the MFMA's 32-row A operand and the (few) tokens its 32-column B operand:
// v_mfma_f32_32x32x16_bf16 computes C[n][t] += W[n][k] X[t][k].
//
// Work split: one workgroup per (expert group, 32 weight rows); its 4 waves
// split the K range; every lane streams 128 contiguous bytes of one weight
// row per step (eight 16-byte loads, prefetched one step ahead), so each
// weight byte is read exactly once and every 128-byte line is consumed by a
// single lane.  The reduction over K runs in the same lane order in both
// operands, so lane l can hold k in [64*(l/32), 64*(l/32)+64) of the step:
// the MFMA sums over whichever 16 k values the two operands hold in common.
// Partial sums of waves 1..3 are reduced into wave 0 through LDS; wave 0 runs
// the epilogue (SwiGLU for the gate/up pair) and writes bf16.
#include "common.h"
#include "ffn_impl.h"

namespace moe {
namespace {

constexpr int kWaves = 4;
constexpr int kStepK = 128;  // K elements per wave step (64 per lane half)

template <int NCH, bool GATED>
struct StepRegs {
  u32x4 w0[8];
  u32x4 w1[GATED ? 8 : 1];
  u32x4 x[NCH][8];
};

template <int NCH, bool GATED>
__device__ __forceinline__ void load_step(StepRegs<NCH, GATED>& r, const GemmArgs& a, int g,
                                          int wrow, bool wrow_ok, int row_base, int tok0, int m,
                                          int kb) {
  const int lane = lane_id();
  const int k_lane = kb * kStepK + (lane >> 5) * 64;  // first k of this lane's slice
  const size_t gbase = static_cast<size_t>(g) * a.group_stride;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int kk = k_lane + 8 * j;
    const bool kok = kk < a.K;
    size_t off = 0;
    if (kok) off = gbase + weight_col_offset(a, kk) + static_cast<size_t>(wrow) * a.ldw;
    const u32x4 zero = {0u, 0u, 0u, 0u};
    r.w0[j] = (kok && wrow_ok) ? load16_nt(a.w0 + off) : zero;
    if constexpr (GATED) r.w1[j] = (kok && wrow_ok) ? load16_nt(a.w1 + off) : zero;
  }
#pragma unroll
  for (int ch = 0; ch < NCH; ++ch) {
    const int tok = tok0 + ch * 32 + (lane & 31);
    const bool tok_ok = tok < m;
    const uint16_t* px = a.x + static_cast<size_t>(row_base + (tok_ok ? tok : 0)) * a.K;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int kk = k_lane + 8 * j;
      const u32x4 zero = {0u, 0u, 0u, 0u};
      r.x[ch][j] = (tok_ok && kk < a.K) ? load16(px + kk) : zero;
    }
  }
}

template <int NCH, bool GATED>
__device__ __forceinline__ void mma_step(const StepRegs<NCH, GATED>& r, f32x16 (&acc0)[NCH],
                                         f32x16 (&acc1)[NCH]) {
#pragma unroll
  for (int j = 0; j < 8; ++j) {
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch) {
      acc0[ch] = mfma32x32x16(as_bf16x8(r.w0[j]), as_bf16x8(r.x[ch][j]), acc0[ch]);
      if constexpr (GATED)
        acc1[ch] = mfma32x32x16(as_bf16x8(r.w1[j]), as_bf16x8(r.x[ch][j]), acc1[ch]);
    }
  }
}

template <int NCH, bool GATED>
__global__ __launch_bounds__(kWaves * kWave) void skinny_kernel(GemmArgs a) {
  constexpr int kMats = GATED ? 2 : 1;
  __shared__ float red[kWaves - 1][kMats][NCH][16][kWave];
  const int g = blockIdx.y;
  int row_base = 0, m = a.static_rows;
  if (a.offsets) {
    row_base = a.offsets[g];
    m = a.offsets[g + 1] - row_base;
  }
  if (m <= 0) return;  // an expert with no rows costs no weight traffic
  const int wave = threadIdx.x / kWave;
  const int lane = lane_id();
  const int n0 = blockIdx.x * 32;
  const int wrow = n0 + (lane & 31);
  const bool wrow_ok = wrow < a.N;
  const int nkb = ceil_div(a.K, kStepK);
  const int kb0 = wave * nkb / kWaves;
  const int kb1 = (wave + 1) * nkb / kWaves;

  for (int tok0 = 0; tok0 < m; tok0 += 32 * NCH) {
    f32x16 acc0[NCH], acc1[NCH];
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch) {
      acc0[ch] = f32x16{};
      acc1[ch] = f32x16{};
    }
    if (kb0 < kb1) {
      StepRegs<NCH, GATED> cur, nxt;
      load_step<NCH, GATED>(cur, a, g, wrow, wrow_ok, row_base, tok0, m, kb0);
      for (int kb = kb0; kb < kb1; ++kb) {
        if (kb + 1 < kb1) load_step<NCH, GATED>(nxt, a, g, wrow, wrow_ok, row_base, tok0, m, kb + 1);
        mma_step<NCH, GATED>(cur, acc0, acc1);
        cur = nxt;
      }
    }
    // reduce the K-split partial sums into wave 0
    if (wave > 0) {
#pragma unroll
      for (int ch = 0; ch < NCH; ++ch)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          red[wave - 1][0][ch][v][lane] = acc0[ch][v];
          if constexpr (GATED) red[wave - 1][kMats - 1][ch][v][lane] = acc1[ch][v];
        }
    }
    __syncthreads();
    if (wave == 0) {
#pragma unroll
      for (int w = 0; w < kWaves - 1; ++w)
#pragma unroll
        for (int ch = 0; ch < NCH; ++ch)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            acc0[ch][v] += red[w][0][ch][v][lane];
            if constexpr (GATED) acc1[ch][v] += red[w][kMats - 1][ch][v][lane];
          }
      // lane holds C[n = 8*(v/4) + 4*(lane/32) + v%4][t = lane%32] of each chunk
#pragma unroll
      for (int ch = 0; ch < NCH; ++ch) {
        const int tok = tok0 + ch * 32 + (lane & 31);
        if (tok >= m) continue;
        uint16_t* orow = a.out + static_cast<size_t>(row_base + tok) * a.N;
#pragma unroll
        for (int v4 = 0; v4 < 4; ++v4) {
          const int n = n0 + 8 * v4 + 4 * (lane >> 5);
          if (n >= a.N) continue;
          float o[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float c0 = acc0[ch][4 * v4 + i];
            o[i] = GATED ? silu(c0) * acc1[ch][4 * v4 + i] : c0;
          }
          uint2 pk;
          pk.x = pack_bf16x2(o[0], o[1]);
          pk.y = pack_bf16x2(o[2], o[3]);
          *reinterpret_cast<uint2*>(orow + n) = pk;
        }
      }
    }
    __syncthreads();
  }
}

template <int NCH, bool GATED>
hipError_t launch_skinny_t(const Segments& seg, const GemmArgs& a, hipStream_t st) {
  dim3 grid(ceil_div(a.N, 32), seg.groups);
  hipLaunchKernelGGL((skinny_kernel<NCH, GATED>), grid, dim3(kWaves * kWave), 0, st, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_skinny(const Segments& seg, const GemmArgs& a, bool gated, hipStream_t st) {
  // chunks of 32 tokens held at once; more rows are handled by re-streaming
  if (seg.max_rows <= 32)
    return gated ? launch_skinny_t<1, true>(seg, a, st) : launch_skinny_t<1, false>(seg, a, st);
  return gated ? launch_skinny_t<2, true>(seg, a, st) : launch_skinny_t<2, false>(seg, a, st);
}

}  // namespace moe
