// Top-k gating and source-aware routing statistics (gfx950).
//
// Selection (Sec. 2.1): a group of G lanes owns one token, each lane holding
// V = ceil(E/G) logits (lane gl holds experts gl, gl+G, ...).  Every logit is
// turned into a 64-bit key whose unsigned order is the selection order:
//   high word: the fp32 bits mapped to an order-preserving unsigned integer
//              (-0.0 folded onto +0.0, every NaN onto 0, below -inf);
//   low word:  ~expert, so equal logits prefer the lower expert index.
// k rounds of a group-wide max over those keys pick the experts in order;
// lane j of the group keeps the j-th pick, then the group computes the gates,
// the softmax of the picked logits renormalised over the k picks.
//
// Statistics (Sec. 5.1, the matrices A_{l,s,e} and B_{l,e}): each block
// counts its pairs into an S x E int32 histogram in LDS and flushes the
// non-zero bins with one 64-bit atomic add each.  Integer atomics make the
// result independent of the order in which blocks land.
#include "common.h"
#include "kernels.h"

namespace moe {
namespace {

constexpr int kBlock = 256;
constexpr int kLdsBinsMax = 16384;  // S*E bins kept in LDS (64 KB)

__device__ __forceinline__ uint32_t order_key(float f) {
  if (f != f) return 0u;            // NaN: below every number
  if (f == 0.0f) f = 0.0f;          // -0.0 ties +0.0
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float key_value(uint32_t key) {
  const uint32_t u = (key & 0x80000000u) ? (key & 0x7fffffffu) : ~key;
  return __uint_as_float(u);
}

__device__ __forceinline__ uint64_t umax64(uint64_t a, uint64_t b) { return a > b ? a : b; }

__device__ __forceinline__ void count_pair(int s, int e, int S, int E, bool use_lds, int* hist,
                                           unsigned long long* counts, int32_t* expert_load) {
  if (s < 0 || s >= S || e < 0 || e >= E) return;
  if (use_lds) {
    atomicAdd(&hist[s * E + e], 1);
  } else {
    atomicAdd(&counts[static_cast<size_t>(s) * E + e], 1ull);
    if (expert_load) atomicAdd(&expert_load[e], 1);
  }
}

__device__ __forceinline__ void flush_hist(const int* hist, int bins, int E,
                                           unsigned long long* counts, int32_t* expert_load) {
  for (int b = threadIdx.x; b < bins; b += blockDim.x) {
    const int c = hist[b];
    if (c) {
      atomicAdd(&counts[b], static_cast<unsigned long long>(c));
      if (expert_load) atomicAdd(&expert_load[b % E], c);
    }
  }
}

template <int G, int V>
__global__ __launch_bounds__(kBlock) void route_kernel(
    int T, int E, int k, int tokens_per_block, const float* __restrict__ logits,
    int32_t* __restrict__ topk_idx, float* __restrict__ topk_w, const int32_t* __restrict__ src,
    int S, unsigned long long* __restrict__ counts, int32_t* __restrict__ expert_load,
    int lds_bins) {
  extern __shared__ int hist[];
  constexpr int kGroups = kBlock / G;
  const bool stats = counts != nullptr;
  const bool use_lds = lds_bins > 0;
  const int tid = threadIdx.x;
  const int gl = tid & (G - 1);
  const int group = tid / G;
  if (stats && use_lds) {
    for (int b = tid; b < lds_bins; b += kBlock) hist[b] = 0;
    __syncthreads();
  }
  const int t0 = blockIdx.x * tokens_per_block;
  const int t1 = min(T, t0 + tokens_per_block);
  for (int base = t0; base < t1; base += kGroups) {
    const int t = base + group;
    const bool valid = t < t1;
    uint64_t key[V];
#pragma unroll
    for (int v = 0; v < V; ++v) {
      const int e = gl + G * v;
      key[v] = 0;
      if (valid && e < E) {
        const float f = logits[static_cast<size_t>(t) * E + e];
        key[v] = (static_cast<uint64_t>(order_key(f)) << 32) | static_cast<uint32_t>(~e);
      }
    }
    uint32_t my_key = 0;
    int my_e = 0;
    for (int r = 0; r < k; ++r) {
      uint64_t best = key[0];
#pragma unroll
      for (int v = 1; v < V; ++v) best = umax64(best, key[v]);
#pragma unroll
      for (int off = G / 2; off > 0; off >>= 1)
        best = umax64(best, __shfl_xor(static_cast<unsigned long long>(best), off, G));
      const int e = static_cast<int>(~static_cast<uint32_t>(best));
#pragma unroll
      for (int v = 0; v < V; ++v)
        if (e == gl + G * v) key[v] = 0;
      if (gl == r) {
        my_key = static_cast<uint32_t>(best >> 32);
        my_e = e;
      }
    }
    const float val = key_value(my_key);
    const float m = __shfl(val, 0, G);
    const float ex = (gl < k) ? expf(val - m) : 0.0f;
    float sum = ex;
#pragma unroll
    for (int off = G / 2; off > 0; off >>= 1) sum += __shfl_xor(sum, off, G);
    if (valid && gl < k) {
      const size_t o = static_cast<size_t>(t) * k + gl;
      topk_idx[o] = my_e;
      topk_w[o] = ex / sum;
      if (stats) count_pair(src[t], my_e, S, E, use_lds, hist, counts, expert_load);
    }
  }
  if (stats && use_lds) {
    __syncthreads();
    flush_hist(hist, lds_bins, E, counts, expert_load);
  }
}

__global__ __launch_bounds__(kBlock) void stats_kernel(int n_pairs, int k, int S, int E,
                                                       int pairs_per_block,
                                                       const int32_t* __restrict__ src,
                                                       const int32_t* __restrict__ topk_idx,
                                                       unsigned long long* __restrict__ counts,
                                                       int32_t* __restrict__ expert_load,
                                                       int lds_bins) {
  extern __shared__ int hist[];
  const bool use_lds = lds_bins > 0;
  if (use_lds) {
    for (int b = threadIdx.x; b < lds_bins; b += kBlock) hist[b] = 0;
    __syncthreads();
  }
  const int p0 = blockIdx.x * pairs_per_block;
  const int p1 = min(n_pairs, p0 + pairs_per_block);
  for (int p = p0 + threadIdx.x; p < p1; p += kBlock)
    count_pair(src[p / k], topk_idx[p], S, E, use_lds, hist, counts, expert_load);
  if (use_lds) {
    __syncthreads();
    flush_hist(hist, lds_bins, E, counts, expert_load);
  }
}

__global__ void fill_i32_kernel(int32_t* p, int n, int32_t value) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = value;
}

template <int G, int V>
hipError_t launch_route_gv(int T, int E, int k, const float* logits, int32_t* topk_idx,
                           float* topk_w, const int32_t* src, int S, int64_t* counts,
                           int32_t* expert_load, hipStream_t st) {
  constexpr int kGroups = kBlock / G;
  // 4 tokens per group and block keeps the histogram flush amortised while
  // leaving enough blocks to fill the chip at the prefill sizes.
  const int tokens_per_block = kGroups * 4;
  const int blocks = ceil_div(T, tokens_per_block);
  const int bins = (counts && S * E <= kLdsBinsMax) ? S * E : 0;
  hipLaunchKernelGGL((route_kernel<G, V>), dim3(blocks), dim3(kBlock), bins * sizeof(int), st, T,
                     E, k, tokens_per_block, logits, topk_idx, topk_w, src, S,
                     reinterpret_cast<unsigned long long*>(counts), expert_load, bins);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_route(int T, int E, int k, const float* logits, int32_t* topk_idx,
                        float* topk_w, const int32_t* src, int S, int64_t* counts,
                        int32_t* expert_load, hipStream_t st) {
  if (T == 0) return hipSuccess;
#define MOE_ROUTE(G, V) \
  return launch_route_gv<G, V>(T, E, k, logits, topk_idx, topk_w, src, S, counts, expert_load, st)
  if (E <= 2) MOE_ROUTE(2, 1);
  if (E <= 4) MOE_ROUTE(4, 1);
  if (E <= 8) MOE_ROUTE(8, 1);
  if (E <= 16) MOE_ROUTE(16, 1);
  if (E <= 32) MOE_ROUTE(32, 1);
  if (E <= 64) MOE_ROUTE(64, 1);
  if (E <= 128) MOE_ROUTE(64, 2);
  if (E <= 256) MOE_ROUTE(64, 4);
  if (E <= 512) MOE_ROUTE(64, 8);
  MOE_ROUTE(64, 16);
#undef MOE_ROUTE
}

hipError_t launch_route_stats(int T, int k, int S, int E, const int32_t* src,
                              const int32_t* topk_idx, int64_t* counts, int32_t* expert_load,
                              hipStream_t st) {
  const int n_pairs = T * k;
  if (n_pairs == 0) return hipSuccess;
  const int pairs_per_block = 2048;
  const int blocks = ceil_div(n_pairs, pairs_per_block);
  const int bins = (S * E <= kLdsBinsMax) ? S * E : 0;
  hipLaunchKernelGGL(stats_kernel, dim3(blocks), dim3(kBlock), bins * sizeof(int), st, n_pairs, k,
                     S, E, pairs_per_block, src, topk_idx,
                     reinterpret_cast<unsigned long long*>(counts), expert_load, bins);
  return hipGetLastError();
}

hipError_t launch_fill_i32(int32_t* p, int n, int32_t value, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(fill_i32_kernel, dim3(ceil_div(n, 256)), dim3(256), 0, st, p, n, value);
  return hipGetLastError();
}

}  // namespace moe
