// Dispatch of the selected (token, expert) pairs to the locally hosted
// experts (Sec. 2.1 dispatch; Sec. 5.2, this GPU's slice of the placement).
//
// A stable counting sort of the T*k pairs by local slot, in three passes
// over tiles of kTile consecutive pairs (token-major order; the second is
// folded into the third when tiles x slots is small, see kInlineScanMax):
//   1. count   per tile and slot, LDS atomics -> tile_counts[tile][slot];
//              in the layer's forward pass also the source x expert
//              statistics of the tile's pairs (Sec. 5.1; over all experts):
//              the tile's LDS histogram is stored as one row, which extra
//              blocks of the scatter launch sum over the tiles (one atomic
//              per bin), or, with too many tiles or bins for that (see
//              stats_bins_per_block), flushed with one global atomic per
//              non-zero bin of the tile;
//   2. scan    one block per slot: exclusive prefix over the tiles (in
//              place) and the slot's total;
//   3. scatter one block of kTile/64 waves per tile, a 64-pair chunk per
//              wave: each pair ORs its lane bit into the chunk's LDS mask
//              of its slot and ranks itself by the popcount of the lower
//              lanes' bits; the chunks of a tile are chained by a per-slot
//              prefix over the waves, so ties keep token order without
//              depending on atomic order.  Each block also derives
//              the slot offsets from the totals (block 0 stores them).
//              Writes perm_token and inv_pos.
// When all pairs fit in one tile (decode-sized batches) a single one-block
// kernel does the three steps.  The row gather x_perm[r] = x[perm_token[r]]
// is a separate, bandwidth-bound kernel that copies 16-byte vectors.
#include "common.h"
#include "dispatch_impl.h"
#include "kernels.h"

#include <algorithm>

namespace moe {
namespace {

constexpr int kTile = kDispatchPairs;  // pairs per tile of the count and scatter passes

// Optionally also the source x expert statistics of the tile's pairs (over
// all E experts, local or not): st.counts != nullptr.
struct PermStats {
  int k, S;
  const int32_t* src;
  unsigned long long* counts;
  int32_t* expert_load;
  int lds_bins;  // S*E bins in LDS after the slot map and slot counts (0: global atomics)
  int32_t* part;  // non-null: the tile's histogram goes to row tile of part (no atomics)
};

// Statistics summed in two levels: the count pass stores each tile's whole
// LDS histogram as a row of part [n_tiles][S*E]; extra blocks of the
// scatter launch, which run beside its tile blocks, each sum bpb bins (a
// power of two) over the rows and add them to the counts with one atomic
// per bin (and to the expert's load B).  A tile's flush instead issues one
// global atomic per non-zero bin, and where many tiles hit the same bins
// those atomics queue on each other.  At most kStatsLoads loads per thread
// (bpb * n_tiles <= kStatsLoads * kTile) and kStatsPartMax ints of rows.
constexpr int kStatsLoads = 8;
constexpr long long kStatsPartMax = 1LL << 22;
struct StatsReduce {
  const int32_t* part;  // nullptr: no reduction blocks
  int bins, bpb, E;
  unsigned long long* counts;
  int32_t* expert_load;
};

// Bins per reduction block, or 0 where the count pass flushes with atomics.
int stats_bins_per_block(int n_tiles, int bins) {
  if (n_tiles < 2 || bins <= 0 || bins > kLdsBinsMax) return 0;
  if (static_cast<long long>(n_tiles) * bins > kStatsPartMax) return 0;
  int bpb = 0;
  for (int b = 1; b <= kTile && static_cast<long long>(b) * n_tiles <= static_cast<long long>(kStatsLoads) * kTile;
       b *= 2)
    bpb = b;
  return bpb;
}

// One reduction block (index rb): bins rb * bpb .. + bpb - 1 of the rows.
// Thread (row t0, bin j) sums rows t0, t0 + kTile / bpb, ...; the lanes of
// a wave that share a bin add up by shuffles, the waves through LDS
// (integer sums: the result does not depend on the order of the adds).
__device__ void stats_reduce_block(const StatsReduce& sr, int n_tiles, int rb, int* red) {
  const int bpb = sr.bpb;
  const int j = threadIdx.x & (bpb - 1), bin = rb * bpb + j;
  const int t0 = threadIdx.x / bpb, dt = kTile / bpb;
  int v[kStatsLoads];
#pragma unroll
  for (int u = 0; u < kStatsLoads; ++u) {
    const int t = t0 + u * dt;
    const bool ok = t < n_tiles && bin < sr.bins;
    v[u] = sr.part[ok ? static_cast<size_t>(t) * sr.bins + bin : 0];
  }
  for (int i = threadIdx.x; i < bpb; i += blockDim.x) red[i] = 0;
  __syncthreads();
  int c = 0;
#pragma unroll
  for (int u = 0; u < kStatsLoads; ++u)
    if (t0 + u * dt < n_tiles && bin < sr.bins) c += v[u];
  for (int off = bpb; off < kWave; off <<= 1) c += __shfl_xor(c, off);
  if (c != 0 && (bpb >= kWave || lane_id() < bpb)) atomicAdd(&red[j], c);
  __syncthreads();
  if (static_cast<int>(threadIdx.x) < bpb && bin < sr.bins) {
    const int total = red[threadIdx.x];
    if (total != 0) {
      atomicAdd(&sr.counts[bin], static_cast<unsigned long long>(total));
      if (sr.expert_load) atomicAdd(&sr.expert_load[bin % sr.E], total);
    }
  }
}

__global__ __launch_bounds__(256) void perm_count_kernel(int n_pairs, int E, int E_local,
                                                         const int32_t* __restrict__ local_experts,
                                                         const int32_t* __restrict__ topk_idx,
                                                         int32_t* __restrict__ tile_counts, PermStats st) {
  extern __shared__ int sm[];
  int* slot_of = sm;
  int* cnt = sm + E;
  int* hist = cnt + E_local;
  const bool stats = st.counts != nullptr;
  const bool use_lds = st.lds_bins > 0;
  for (int s = threadIdx.x; s < E_local; s += blockDim.x) cnt[s] = 0;
  if (stats && use_lds)
    for (int b = threadIdx.x; b < st.lds_bins; b += blockDim.x) hist[b] = 0;
  // a thread's pairs of the tile: every load goes out first, beside the
  // slot map's (pairs past the end read pair 0 and are dropped)
  constexpr int kPer = kTile / 256;
  const int p0 = blockIdx.x * kTile + threadIdx.x;
  int e[kPer], src[kPer];
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    const int p = p0 + i * 256;
    const int pc = p < n_pairs ? p : 0;
    e[i] = topk_idx[pc];
    src[i] = stats ? st.src[pc / st.k] : 0;
  }
  build_slot_map(slot_of, E, E_local, local_experts);  // (ends with a barrier)
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    if (p0 + i * 256 >= n_pairs) break;
    const int s = slot_lookup(slot_of, e[i], E);
    if (s >= 0) atomicAdd(&cnt[s], 1);
    if (stats) count_pair(src[i], e[i], st.S, E, use_lds, hist, st.counts, st.expert_load);
  }
  __syncthreads();
  for (int s = threadIdx.x; s < E_local; s += blockDim.x)
    tile_counts[static_cast<size_t>(blockIdx.x) * E_local + s] = cnt[s];
  if (stats && use_lds) {
    if (st.part != nullptr) {
      int32_t* row = st.part + static_cast<size_t>(blockIdx.x) * st.lds_bins;
      for (int b = threadIdx.x; b < st.lds_bins; b += blockDim.x) row[b] = hist[b];
    } else {
      flush_hist(hist, st.lds_bins, E, st.counts, st.expert_load);
    }
  }
}


__global__ __launch_bounds__(256) void perm_scan_kernel(int n_tiles, int E_local,
                                                        int32_t* __restrict__ tile_counts,
                                                        int32_t* __restrict__ slot_total) {
  const int s = blockIdx.x;
  int carry = 0;
  for (int t0 = 0; t0 < n_tiles; t0 += blockDim.x) {
    const int t = t0 + threadIdx.x;
    const size_t i = static_cast<size_t>(t) * E_local + s;
    const int v = t < n_tiles ? tile_counts[i] : 0;
    int total;
    const int ex = block_exclusive_scan(v, &total);
    if (t < n_tiles) tile_counts[i] = carry + ex;
    carry += total;
  }
  if (threadIdx.x == 0) slot_total[s] = carry;
}

constexpr int kScatterWaves = kTile / kWave;
// largest tiles x slots whose counts every scatter block sums itself (64
// KB): with four slots per 16-byte load, a thread then has at most
// kInlineLoads loads (tiles x slots / (4 kTile)), all in flight at once
constexpr int kInlineLoads = 8;
constexpr long long kInlineScanMax = 4LL * kTile * kInlineLoads;

// inline_scan: tile_prefix holds the count pass's raw per-tile counts (no
// scan pass ran); each block sums, per slot, the counts of the tiles before
// its own and of all tiles itself (E_local a multiple of 4, at most
// 4 kTile).  Else tile_prefix and slot_total come from the scan pass.
// RED: blocks past the tiles sum the statistics (see StatsReduce); without
// it the kernel has no such branch.
template <bool RED>
__global__ __launch_bounds__(kTile) void perm_scatter_kernel(
    int n_pairs, int k, int E, int E_local, const int32_t* __restrict__ local_experts,
    const int32_t* __restrict__ topk_idx, const int32_t* __restrict__ tile_prefix,
    const int32_t* __restrict__ slot_total, int32_t* __restrict__ offsets,
    int32_t* __restrict__ perm_token, int32_t* __restrict__ inv_pos, bool inline_scan, StatsReduce sr) {
  extern __shared__ int sm[];
  if constexpr (RED) {
    // the tile blocks' arguments are read here, before the branch on the
    // block's role: the compiler would otherwise fetch them only past it,
    // one more round trip to the argument segment before the first load
    asm volatile("" ::"s"(k), "s"(E), "s"(E_local), "s"(local_experts), "s"(topk_idx), "s"(tile_prefix),
                 "s"(slot_total), "s"(offsets), "s"(perm_token), "s"(inv_pos), "s"(static_cast<int>(inline_scan)));
    if (static_cast<int>(blockIdx.x) >= ceil_div(n_pairs, kTile)) {
      stats_reduce_block(sr, ceil_div(n_pairs, kTile), blockIdx.x - ceil_div(n_pairs, kTile), sm);
      return;
    }
  }
  // [wave][slot]: bit l set when lane l of the wave's chunk has the slot
  uint64_t* mask = reinterpret_cast<uint64_t*>(sm);
  int* part = sm + 2 * kScatterWaves * E_local;  // inline scan: [2][rows][slot] partial sums
  int* slot_of = part + (inline_scan ? 8 * kTile : 0);
  int* base = slot_of + E;             // first row of each slot for this tile
  int* cnt = base + E_local;           // [wave][slot]: rows of the slot in earlier chunks
  const int tile = blockIdx.x;
  const int n_tiles = ceil_div(n_pairs, kTile);
  const int wave = threadIdx.x / kWave, lane = lane_id();
  // the pair's expert id is loaded first, beside the slot map's loads
  const int p = tile * kTile + wave * kWave + lane;
  const int e_p = topk_idx[p < n_pairs ? p : 0];
  for (int i = threadIdx.x; i < kScatterWaves * E_local; i += blockDim.x) mask[i] = 0;
  if (inline_scan) {
    // thread (row r, slots 4 sl .. 4 sl + 3) sums tiles r, r + R, ... (R
    // rows of E_local / 4 threads), 16 bytes per load, one batch of loads
    // (see kInlineLoads); rows then add up through LDS
    const int W = E_local / 4;
    const int R = kTile / W;
    const int r = threadIdx.x / W, sl = threadIdx.x - r * W;
    int4 before = {0, 0, 0, 0}, all = {0, 0, 0, 0};
    if (r < R) {
      for (int t0 = r; t0 < n_tiles; t0 += kInlineLoads * R) {
        int4 v[kInlineLoads];
#pragma unroll
        for (int u = 0; u < kInlineLoads; ++u) {
          const int tt = t0 + u * R;
          v[u] = *reinterpret_cast<const int4*>(tile_prefix + static_cast<size_t>(tt < n_tiles ? tt : 0) * E_local +
                                                4 * sl);
        }
#pragma unroll
        for (int u = 0; u < kInlineLoads; ++u) {
          const int tt = t0 + u * R;
          const int4 c = tt < n_tiles ? v[u] : int4{0, 0, 0, 0};
          all.x += c.x; all.y += c.y; all.z += c.z; all.w += c.w;
          if (tt < tile) {
            before.x += c.x; before.y += c.y; before.z += c.z; before.w += c.w;
          }
        }
      }
      *reinterpret_cast<int4*>(part + r * E_local + 4 * sl) = before;
      *reinterpret_cast<int4*>(part + (R + r) * E_local + 4 * sl) = all;
    }
  }
  build_slot_map(slot_of, E, E_local, local_experts);  // (ends with a barrier)
  // slot offsets: exclusive scan of the totals
  int carry = 0;
  for (int s0 = 0; s0 < E_local; s0 += blockDim.x) {
    const int s = s0 + threadIdx.x;
    int tot = 0, pre = 0;
    if (s < E_local) {
      if (inline_scan) {
        const int R = kTile / (E_local / 4);
        for (int r = 0; r < R; ++r) {
          pre += part[r * E_local + s];
          tot += part[(R + r) * E_local + s];
        }
      } else {
        tot = slot_total[s];
        pre = tile_prefix[static_cast<size_t>(tile) * E_local + s];
      }
    }
    int total;
    const int ex = block_exclusive_scan(tot, &total);
    if (s < E_local) {
      base[s] = carry + ex + pre;
      if (tile == 0) offsets[s] = carry + ex;
    }
    carry += total;
  }
  if (tile == 0 && threadIdx.x == 0) offsets[E_local] = carry;
  // each pair sets its lane's bit in its chunk's mask of its slot: an OR, so
  // the masks do not depend on the order the lanes' updates land in; a
  // pair's rank in its chunk is then the count of lower lanes in its mask
  int s = -1;
  if (p < n_pairs) {
    s = slot_lookup(slot_of, e_p, E);
    if (s < 0) inv_pos[p] = -1;
  }
  if (s >= 0) atomicOr(reinterpret_cast<unsigned long long*>(&mask[wave * E_local + s]), 1ull << lane);
  __syncthreads();
  for (int sl = threadIdx.x; sl < E_local; sl += blockDim.x) {
    int run = 0;
    for (int w = 0; w < kScatterWaves; ++w) {
      cnt[w * E_local + sl] = run;
      run += __popcll(mask[w * E_local + sl]);
    }
  }
  __syncthreads();
  if (s >= 0) {
    const uint64_t below = (1ull << lane) - 1ull;
    const int rank = __popcll(mask[wave * E_local + s] & below);
    const int pos = base[s] + cnt[wave * E_local + s] + rank;
    perm_token[pos] = p / k;
    inv_pos[p] = pos;
  }
}

// All three steps for n_pairs <= kTile in one block of 1024 threads.
__global__ __launch_bounds__(1024) void perm_single_kernel(int n_pairs, int k, int E, int E_local,
                                                           const int32_t* __restrict__ local_experts,
                                                           const int32_t* __restrict__ topk_idx,
                                                           int32_t* __restrict__ offsets,
                                                           int32_t* __restrict__ perm_token,
                                                           int32_t* __restrict__ inv_pos) {
  extern __shared__ int sm[];
  // the expert ids into LDS in one pass (n_pairs <= kTile < blockDim.x)
  int* ids = sm + dispatch_one_block_ints(E, E_local);
  if (static_cast<int>(threadIdx.x) < n_pairs) ids[threadIdx.x] = topk_idx[threadIdx.x];
  __syncthreads();
  dispatch_one_block(n_pairs, k, E, E_local, local_experts, ids, offsets, perm_token, inv_pos, sm);
}

__global__ __launch_bounds__(256) void gather_rows_kernel(int H, const int32_t* __restrict__ perm_token,
                                                          const int32_t* __restrict__ n_rows,
                                                          const uint16_t* __restrict__ x,
                                                          uint16_t* __restrict__ x_perm) {
  const int R = *n_rows;
  const int vpr = H / 8;  // 16-byte vectors per row
  const int lane = lane_id();
  const int n_waves = gridDim.x * (blockDim.x / kWave);
  for (int r = blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave; r < R; r += n_waves) {
    const uint16_t* src = x + static_cast<size_t>(perm_token[r]) * H;
    uint16_t* dst = x_perm + static_cast<size_t>(r) * H;
    for (int v = lane; v < vpr; v += kWave) store16(dst + v * 8, load16(src + v * 8));
  }
}

}  // namespace

size_t permute_ws_bytes(int T, int k, int E_local, int S, int E) {
  const int n_tiles = ceil_div(T * k, kTile);
  // tile counts, slot totals
  size_t bytes = (static_cast<size_t>(n_tiles) + 1) * static_cast<size_t>(E_local) * sizeof(int32_t);
  // the statistics' per-tile rows, where they are summed in two levels
  if (stats_bins_per_block(n_tiles, S * E) > 0)
    bytes += static_cast<size_t>(n_tiles) * static_cast<size_t>(S * E) * sizeof(int32_t);
  return bytes;
}

hipError_t launch_permute(int T, int k, int E, int E_local, const int32_t* local_experts,
                          const int32_t* topk_idx, int32_t* offsets, int32_t* perm_token,
                          int32_t* inv_pos, void* ws, hipStream_t st, const int32_t* src, int S,
                          int64_t* counts, int32_t* expert_load) {
  const int n_pairs = T * k;
  if (counts != nullptr && n_pairs <= kTile) return hipErrorInvalidValue;  // no count pass to take them
  if (n_pairs == 0) return launch_fill_i32(offsets, E_local + 1, 0, st);
  const int n_tiles = ceil_div(n_pairs, kTile);
  int32_t* tile_counts = static_cast<int32_t*>(ws);
  if (n_tiles == 1) {
    const size_t lds = static_cast<size_t>(dispatch_one_block_ints(E, E_local) + kTile) * sizeof(int);
    hipLaunchKernelGGL(perm_single_kernel, dim3(1), dim3(1024), lds, st, n_pairs, k, E, E_local,
                       local_experts, topk_idx, offsets, perm_token, inv_pos);
    return hipGetLastError();
  }
  PermStats ps{k, S, src, reinterpret_cast<unsigned long long*>(counts), expert_load, 0, nullptr};
  if (counts != nullptr && S * E <= kLdsBinsMax) ps.lds_bins = S * E;
  StatsReduce sr{nullptr, 0, 0, E, ps.counts, expert_load};
  int n_red = 0;  // reduction blocks after the tile blocks of the scatter launch
  if (counts != nullptr) {
    const int bpb = stats_bins_per_block(n_tiles, S * E);
    if (bpb > 0) {
      ps.part = tile_counts + (static_cast<size_t>(n_tiles) + 1) * E_local;
      sr = StatsReduce{ps.part, S * E, bpb, E, ps.counts, expert_load};
      n_red = ceil_div(S * E, bpb);
    }
  }
  const size_t lds_count = static_cast<size_t>(E + E_local + ps.lds_bins) * sizeof(int);
  static unsigned long long lds_set = 0;  // devices with the LDS limit raised
  hipError_t err = set_max_dynamic_lds(reinterpret_cast<const void*>(&perm_count_kernel),
                                       static_cast<int>((2 * kMaxExperts + kLdsBinsMax) * sizeof(int)), &lds_set);
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL(perm_count_kernel, dim3(n_tiles), dim3(256), lds_count, st, n_pairs, E, E_local,
                     local_experts, topk_idx, tile_counts, ps);
  err = hipGetLastError();
  if (err != hipSuccess) return err;
  int32_t* slot_total = tile_counts + static_cast<size_t>(n_tiles) * E_local;
  // few tiles x slots: each scatter block sums the counts it needs itself,
  // which saves the scan launch
  const bool inline_scan = E_local % 4 == 0 && E_local <= 4 * kTile &&
                           static_cast<long long>(n_tiles) * E_local <= kInlineScanMax;
  if (!inline_scan) {
    hipLaunchKernelGGL(perm_scan_kernel, dim3(E_local), dim3(256), 0, st, n_tiles, E_local, tile_counts, slot_total);
    err = hipGetLastError();
    if (err != hipSuccess) return err;
  }
  const size_t lds_scatter =
      static_cast<size_t>(E + (1 + 3 * kScatterWaves) * E_local + (inline_scan ? 8 * kTile : 0)) * sizeof(int);
  static unsigned long long lds_set_scatter[2] = {0, 0};  // devices with the LDS limit raised, per variant
  const bool red = n_red > 0;
  err = set_max_dynamic_lds(red ? reinterpret_cast<const void*>(&perm_scatter_kernel<true>)
                                : reinterpret_cast<const void*>(&perm_scatter_kernel<false>),
                            static_cast<int>((kMaxExperts + (1 + 3 * kScatterWaves) * kMaxExperts + 8 * kTile) *
                                             sizeof(int)),
                            &lds_set_scatter[red ? 1 : 0]);
  if (err != hipSuccess) return err;
  const size_t lds = std::max(lds_scatter, static_cast<size_t>(sr.bpb) * sizeof(int));
  if (red)
    hipLaunchKernelGGL(perm_scatter_kernel<true>, dim3(n_tiles + n_red), dim3(kTile), lds, st, n_pairs, k, E,
                       E_local, local_experts, topk_idx, tile_counts, slot_total, offsets, perm_token, inv_pos,
                       inline_scan, sr);
  else
    hipLaunchKernelGGL(perm_scatter_kernel<false>, dim3(n_tiles), dim3(kTile), lds, st, n_pairs, k, E, E_local,
                       local_experts, topk_idx, tile_counts, slot_total, offsets, perm_token, inv_pos, inline_scan,
                       sr);
  return hipGetLastError();
}

hipError_t launch_gather_rows(int capacity, int H, const int32_t* perm_token, const int32_t* n_rows,
                              const uint16_t* x, uint16_t* x_perm, hipStream_t st) {
  if (capacity == 0) return hipSuccess;
  const int waves_per_block = 4;
  const int blocks = min(ceil_div(capacity, waves_per_block), 4096);
  hipLaunchKernelGGL(gather_rows_kernel, dim3(blocks), dim3(waves_per_block * kWave), 0, st, H,
                     perm_token, n_rows, x, x_perm);
  return hipGetLastError();
}

}  // namespace moe
