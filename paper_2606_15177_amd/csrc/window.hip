// Diagnostics of a profiling window under a placement: the traffic each
// source sends to experts outside its own rank (the cross-DP-group share of
// Sec. 2.2, Fig. 4), the token load of each rank's experts, and the MoE
// pressure of each DP engine (Sec. 4.1: the token-equivalent expert load of
// its ranks, relative to the average engine).
//
// window_layer_kernel: one workgroup per layer.  The placement row is staged
// in LDS; every thread adds its experts' loads into per-rank LDS counters;
// then each wave takes a source and walks its row of A with coalesced loads.
// window_pressure_kernel: one workgroup sums the rank loads of all layers per
// engine and normalises.  Every sum is an integer, so the results do not
// depend on the order in which lanes or atomics land.
#include "common.h"
#include "kernels.h"

namespace moe {
namespace {

constexpr int kWinThreads = 256;
constexpr int kWinWaves = kWinThreads / kWave;

__device__ __forceinline__ int64_t wave_sum_i64(int64_t v) {
  for (int off = kWave / 2; off > 0; off >>= 1) v += __shfl_xor(v, off);
  return v;
}

__global__ __launch_bounds__(kWinThreads) void window_layer_kernel(WindowArgs a) {
  __shared__ int32_t xs[kWindowMaxExperts];
  __shared__ unsigned long long load[kWindowMaxRanks];
  const int l = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int S = a.S, E = a.E, G = a.G;
  const int64_t* A_l = a.A + static_cast<size_t>(l) * S * E;

  for (int g = tid; g < G; g += kWinThreads) load[g] = 0ull;
  for (int e = tid; e < E; e += kWinThreads) xs[e] = a.x[static_cast<size_t>(l) * E + e];
  __syncthreads();

  for (int e = tid; e < E; e += kWinThreads) {
    int64_t b;
    if (a.B) {
      b = a.B[static_cast<size_t>(l) * E + e];
    } else {
      b = 0;
      for (int s = 0; s < S; ++s) b += A_l[static_cast<size_t>(s) * E + e];
    }
    const int g = xs[e];
    if (g >= 0 && g < G) atomicAdd(&load[g], static_cast<unsigned long long>(b));
  }

  for (int s = wave; s < S; s += kWinWaves) {
    const int home = a.home[s];
    const bool home_ok = home >= 0 && home < G;
    const int64_t* row = A_l + static_cast<size_t>(s) * E;
    int64_t tot = 0, rem = 0;
    for (int e = lane; e < E; e += kWave) {
      const int64_t c = row[e];
      tot += c;
      rem += (!home_ok || xs[e] != home) ? c : 0;
    }
    tot = wave_sum_i64(tot);
    rem = wave_sum_i64(rem);
    if (lane == 0) {
      a.total[static_cast<size_t>(l) * S + s] = tot;
      a.remote[static_cast<size_t>(l) * S + s] = rem;
    }
  }
  __syncthreads();
  for (int g = tid; g < G; g += kWinThreads)
    a.rank_load[static_cast<size_t>(l) * G + g] = static_cast<int64_t>(load[g]);
}

__global__ __launch_bounds__(kWinThreads) void window_pressure_kernel(WindowArgs a) {
  __shared__ unsigned long long eng[kWindowMaxEngines];
  __shared__ int64_t all_s;
  const int tid = threadIdx.x;
  const int G = a.G, D = a.n_engines;
  for (int d = tid; d < D; d += kWinThreads) eng[d] = 0ull;
  __syncthreads();
  const size_t n = static_cast<size_t>(a.L) * G;
  for (size_t i = tid; i < n; i += kWinThreads) {
    const int g = static_cast<int>(i % G);
    const int d = a.engine ? a.engine[g] : g;
    if (d >= 0 && d < D) atomicAdd(&eng[d], static_cast<unsigned long long>(a.rank_load[i]));
  }
  __syncthreads();
  if (tid == 0) {
    int64_t all = 0;
    for (int d = 0; d < D; ++d) all += static_cast<int64_t>(eng[d]);
    all_s = all;
  }
  __syncthreads();
  const int64_t all = all_s;
  const double mean = static_cast<double>(all) / D;
  for (int d = tid; d < D; d += kWinThreads)
    a.pressure[d] = all == 0 ? 0.0 : static_cast<double>(static_cast<int64_t>(eng[d])) / mean;
}

}  // namespace

hipError_t launch_window(const WindowArgs& a, hipStream_t st) {
  if (a.L > 0) {
    hipLaunchKernelGGL(window_layer_kernel, dim3(a.L), dim3(kWinThreads), 0, st, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (a.pressure) {
    hipLaunchKernelGGL(window_pressure_kernel, dim3(1), dim3(kWinThreads), 0, st, a);
    return hipGetLastError();
  }
  return hipSuccess;
}

}  // namespace moe
