// Device helpers of the dispatch (the stable counting sort of the selected
// (token, expert) pairs by local slot), shared by the permute kernels and
// the routing kernel's one-block dispatch for decode-sized batches.
#pragma once

#include "common.h"
#include "kernels.h"

namespace moe {

// Source x expert statistics (Sec. 5.1, the matrices A_{l,s,e} and B_{l,e}):
// a block counts its pairs into an S x E int32 histogram in LDS when it has
// at most kLdsBinsMax bins (else straight into the global counts) and then
// flushes the non-zero bins with one 64-bit atomic add each.  Integer
// atomics make the result independent of the order in which blocks land.
constexpr int kLdsBinsMax = 16384;  // S*E bins kept in LDS (64 KB)

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

// slot_of[e] = local slot hosting expert e, or -1.  An expert listed twice
// (outside the documented contract) resolves to its lowest slot, the same in
// every kernel, so the count and scatter passes always agree.  Ends with a
// barrier.
__device__ inline void build_slot_map(int* slot_of, int E, int E_local, const int32_t* local_experts) {
  if (local_experts == nullptr) {
    for (int e = threadIdx.x; e < E; e += blockDim.x) slot_of[e] = e;
  } else {
    for (int e = threadIdx.x; e < E; e += blockDim.x) slot_of[e] = E_local;
    __syncthreads();
    for (int s = threadIdx.x; s < E_local; s += blockDim.x) {
      const int e = local_experts[s];
      if (e >= 0 && e < E) atomicMin(&slot_of[e], s);
    }
    __syncthreads();
    for (int e = threadIdx.x; e < E; e += blockDim.x)
      if (slot_of[e] >= E_local) slot_of[e] = -1;
  }
  __syncthreads();
}

__device__ __forceinline__ int slot_lookup(const int* slot_of, int e, int E) {
  return (e >= 0 && e < E) ? slot_of[e] : -1;
}

// Exclusive scan of one value per thread over a block of blockDim.x threads
// (a multiple of 64, at most 1024).  Returns the exclusive prefix; *total
// receives the block sum.  Ends with a barrier.
__device__ inline int block_exclusive_scan(int v, int* total) {
  __shared__ int wsum[16];
  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
  int inc = v;
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const int o = __shfl_up(inc, off);
    if (lane >= off) inc += o;
  }
  if (lane == kWave - 1) wsum[wave] = inc;
  __syncthreads();
  if (wave == 0) {
    const int n_waves = blockDim.x / kWave;
    int w = lane < n_waves ? wsum[lane] : 0;
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) {
      const int o = __shfl_up(w, off);
      if (lane >= off) w += o;
    }
    if (lane < n_waves) wsum[lane] = w;  // inclusive over waves
  }
  __syncthreads();
  const int before = wave > 0 ? wsum[wave - 1] : 0;
  *total = wsum[blockDim.x / kWave - 1];
  __syncthreads();
  return before + inc - v;
}

// LDS ints that dispatch_one_block takes: the slot map, the slot offsets and
// the per-chunk slot counts.
constexpr int kDispatchChunks = kDispatchPairs / kWave;
__host__ __device__ constexpr int dispatch_one_block_ints(int E, int E_local) {
  return E + (1 + kDispatchChunks) * E_local;
}

// The whole dispatch of n_pairs <= kDispatchPairs pairs by one block of at
// least kDispatchPairs / 2 threads (E_local <= blockDim.x): per-slot
// offsets [E_local + 1], then perm_token and inv_pos in token order within
// each slot.  sm: dispatch_one_block_ints(E, E_local) ints of LDS; ids: the
// pairs' expert ids, already in LDS (the caller stages them; a barrier must
// separate their writes from this call).  Wave w ranks the pairs of 64-pair
// chunks w, w + waves (at most two) by ballot + popcount, and a per-slot
// prefix over the chunks chains them, so ties keep token order without
// depending on atomic order.
__device__ inline void dispatch_one_block(int n_pairs, int k, int E, int E_local,
                                          const int32_t* __restrict__ local_experts, const int* ids,
                                          int32_t* __restrict__ offsets, int32_t* __restrict__ perm_token,
                                          int32_t* __restrict__ inv_pos, int* sm) {
  constexpr int kMaxChunksPerWave = 2;
  int* slot_of = sm;
  int* base = sm + E;           // per slot: total, then first row
  int* ccnt = base + E_local;   // [chunk][slot]: chunk counts, then prefix over chunks
  const int n_chunks = ceil_div(n_pairs, kWave);
  const int n_waves = blockDim.x / kWave;
  const int wave = threadIdx.x / kWave, lane = lane_id();
  for (int i = threadIdx.x; i < n_chunks * E_local; i += blockDim.x) ccnt[i] = 0;
  build_slot_map(slot_of, E, E_local, local_experts);  // (ends with a barrier)
  const uint64_t below = (1ull << lane) - 1ull;
  int slot[kMaxChunksPerWave], rank[kMaxChunksPerWave];
#pragma unroll
  for (int j = 0; j < kMaxChunksPerWave; ++j) {
    const int c = wave + j * n_waves;
    const int p = c * kWave + lane;
    int s = -1;
    if (c < n_chunks && p < n_pairs) {
      s = slot_lookup(slot_of, ids[p], E);
      if (s < 0) inv_pos[p] = -1;
    }
    int r = 0;
    uint64_t pending = __ballot(s >= 0);
    while (pending) {
      const int leader = __ffsll(static_cast<long long>(pending)) - 1;
      const int sl = __shfl(s, leader);
      const uint64_t same = __ballot(s == sl);
      if (s == sl) r = __popcll(same & below);
      if (lane == leader) ccnt[c * E_local + sl] = __popcll(same);
      pending &= ~same;
    }
    slot[j] = s;
    rank[j] = r;
  }
  __syncthreads();
  // per slot: prefix over the chunks, and the slot's total
  for (int sl = threadIdx.x; sl < E_local; sl += blockDim.x) {
    int run = 0;
    for (int c = 0; c < n_chunks; ++c) {
      const int v = ccnt[c * E_local + sl];
      ccnt[c * E_local + sl] = run;
      run += v;
    }
    base[sl] = run;
  }
  __syncthreads();
  const int own = threadIdx.x < E_local ? base[threadIdx.x] : 0;
  int total;
  const int excl = block_exclusive_scan(own, &total);  // (ends with a barrier)
  if (threadIdx.x < E_local) {
    offsets[threadIdx.x] = excl;
    base[threadIdx.x] = excl;
  }
  if (threadIdx.x == 0) offsets[E_local] = total;
  __syncthreads();
#pragma unroll
  for (int j = 0; j < kMaxChunksPerWave; ++j) {
    const int c = wave + j * n_waves;
    const int p = c * kWave + lane;
    if (slot[j] >= 0) {
      const int pos = base[slot[j]] + ccnt[c * E_local + slot[j]] + rank[j];
      perm_token[pos] = p / k;
      inv_pos[p] = pos;
    }
  }
}

}  // namespace moe
