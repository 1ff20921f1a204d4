// Weighted combine back to token order (Sec. 2.1: expert outputs are
// combined and returned):
//   out[t] = sum_{j<k, inv_pos[t*k+j] >= 0} w[t][j] * y_perm[inv_pos[t*k+j]] + y_shared[t]
// One wave per (token, 64 consecutive 16-byte column vectors of its row), so
// that even a decode-sized batch spreads over the whole chip; each lane owns
// one vector and accumulates in fp32, j ascending then the shared term, so
// the result does not depend on scheduling.  Bandwidth-bound: every byte of
// y_perm and y_shared is read once.
#include "common.h"
#include "kernels.h"

namespace moe {
namespace {

constexpr int kMaxK = 32;
constexpr int kLoadsInFlight = 8;  // row loads a lane issues before it accumulates

__global__ __launch_bounds__(256) void combine_kernel(int T, int k, int H,
                                                      const uint16_t* __restrict__ y_perm,
                                                      const int32_t* __restrict__ inv_pos,
                                                      const float* __restrict__ topk_w,
                                                      const uint16_t* __restrict__ y_shared,
                                                      uint16_t* __restrict__ out) {
  const int lane = lane_id();
  const long long n_waves = static_cast<long long>(gridDim.x) * (blockDim.x / kWave);
  const int vpr = H / 8;
  const int chunks = ceil_div(vpr, kWave);
  const long long n_items = static_cast<long long>(T) * chunks;
  for (long long item = static_cast<long long>(blockIdx.x) * (blockDim.x / kWave) + threadIdx.x / kWave;
       item < n_items; item += n_waves) {
    const int t = static_cast<int>(item / chunks);
    const int v0 = static_cast<int>(item - static_cast<long long>(t) * chunks) * kWave;
    // the token's k (row, weight) pairs
    int pos = -1;
    float w = 0.0f;
    if (lane < k) {
      pos = inv_pos[static_cast<size_t>(t) * k + lane];
      w = topk_w[static_cast<size_t>(t) * k + lane];
    }
    // every lane takes part in the shuffles; lanes past the end of the row
    // only skip the memory work
    {
      const int v = v0 + lane;
      const bool active = v < vpr;
      float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
      // eight rows' loads are issued before the first of them is consumed;
      // the sum still runs in j order, and a pair without a local row adds
      // nothing (not even 0 * its gate)
      for (int j0 = 0; j0 < k; j0 += kLoadsInFlight) {
        int r[kLoadsInFlight];
        u32x4 q[kLoadsInFlight];
#pragma unroll
        for (int jj = 0; jj < kLoadsInFlight; ++jj) {
          r[jj] = j0 + jj < k ? __builtin_amdgcn_readlane(pos, j0 + jj) : -1;   // wave-uniform
          q[jj] = (r[jj] >= 0 && active) ? load16(y_perm + static_cast<size_t>(r[jj]) * H + v * 8) : u32x4{0, 0, 0, 0};
        }
#pragma unroll
        for (int jj = 0; jj < kLoadsInFlight; ++jj) {
          const float wj = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(w), j0 + jj < k ? j0 + jj : 0));
          if (r[jj] < 0) continue;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            acc[2 * e] = fmaf(wj, __uint_as_float(q[jj][e] << 16), acc[2 * e]);
            acc[2 * e + 1] = fmaf(wj, __uint_as_float(q[jj][e] & 0xffff0000u), acc[2 * e + 1]);
          }
        }
      }
      if (!active) continue;
      if (y_shared) {
        const u32x4 q = load16(y_shared + static_cast<size_t>(t) * H + v * 8);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          acc[2 * e] += __uint_as_float(q[e] << 16);
          acc[2 * e + 1] += __uint_as_float(q[e] & 0xffff0000u);
        }
      }
      u32x4 o;
#pragma unroll
      for (int e = 0; e < 4; ++e) o[e] = pack_bf16x2(acc[2 * e], acc[2 * e + 1]);
      store16(out + static_cast<size_t>(t) * H + v * 8, o);
    }
  }
}

}  // namespace

hipError_t launch_combine(int T, int k, int H, const uint16_t* y_perm, const int32_t* inv_pos,
                          const float* topk_w, const uint16_t* y_shared, uint16_t* out,
                          hipStream_t st) {
  if (T == 0) return hipSuccess;
  if (k > kMaxK) return hipErrorInvalidValue;
  const int waves_per_block = 4;
  const long long items = static_cast<long long>(T) * ceil_div(H / 8, kWave);
  const int blocks = static_cast<int>(std::min<long long>((items + waves_per_block - 1) / waves_per_block, 8192));
  hipLaunchKernelGGL(combine_kernel, dim3(blocks), dim3(waves_per_block * kWave), 0, st, T, k, H,
                     y_perm, inv_pos, topk_w, y_shared, out);
  return hipGetLastError();
}

}  // namespace moe
