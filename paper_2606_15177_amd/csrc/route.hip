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
// Gating variants (the EXT instantiations): the selection value may instead be
// a sigmoid score s = sigma(l), evaluated in fp64 and rounded to fp32, plus a
// selection-only bias; gates may be the full softmax over all E logits or the
// picked sigmoid scores renormalised; all gates may be scaled.  Under a group
// limit the token's selection values are staged in LDS, lane q of the group
// sums the two first values of expert group q, topk_group rounds of a max
// over those sums keep groups, and the experts of the other groups drop out of
// the selection (key 0, below every kept expert, NaN included).
//
// Decode-sized batches (at most 512 pairs, four token groups): one block
// routes the whole batch and then writes its dispatch (offsets, perm_token,
// inv_pos) as the permute kernels would, saving a launch.
//
// Statistics (Sec. 5.1, the matrices A_{l,s,e} and B_{l,e}): each block
// counts its pairs into an S x E histogram (see count_pair).  A route block
// holds few tokens, so each flushes about one global atomic per pair; the
// layer's forward pass therefore counts in the dispatch's count pass, whose
// blocks hold 512 pairs, whenever that pass runs.
#include "common.h"
#include "dispatch_impl.h"
#include "kernels.h"

namespace moe {
namespace {

constexpr int kBlock = 256;
constexpr int kStatsPairs = 2048;   // (token, expert) pairs per block of the counting kernel

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

struct RouteKernelArgs {
  int T, E, k, tokens_per_block;
  const float* logits;
  int32_t* topk_idx;
  float* topk_w;
  const int32_t* src;
  int S;
  unsigned long long* counts;
  int32_t* expert_load;
  int lds_bins;          // S*E histogram bins in LDS (0: global atomics)
  // gating variant
  int gate;              // 0 softmax over the picks, 1 full softmax, 2 sigmoid
  const float* bias;     // [E] selection-only bias (gate 2), nullable
  float scale;           // gates are multiplied by this
  int n_group, topk_group;  // group limit when n_group > 1
  // the dispatch in the same launch (one block routes the whole batch)
  bool disp;
  DispatchArgs d;
};

__device__ __forceinline__ float sigmoid_score(float l) {
  return static_cast<float>(1.0 / (1.0 + exp(-static_cast<double>(l))));
}

// Butterfly levels within a 16-lane row by DPP (quad swaps, then the half-row
// and row mirrors), across rows by ds_bpermute.  Max and sum are symmetric,
// so after the levels every lane of a G-lane group holds the group's result.
template <int CTRL>
__device__ __forceinline__ int dpp_i32(int v) {
  return __builtin_amdgcn_update_dpp(v, v, CTRL, 0xf, 0xf, false);
}
constexpr int kDppSwap1 = 0xB1;       // quad_perm [1, 0, 3, 2]
constexpr int kDppSwap2 = 0x4E;       // quad_perm [2, 3, 0, 1]
constexpr int kDppHalfMirror = 0x141;  // lane i <-> 7 - i within 8 lanes
constexpr int kDppMirror = 0x140;      // lane i <-> 15 - i within 16 lanes

template <int CTRL>
__device__ __forceinline__ uint64_t dpp_u64(uint64_t v) {
  const int lo = dpp_i32<CTRL>(static_cast<int>(static_cast<uint32_t>(v)));
  const int hi = dpp_i32<CTRL>(static_cast<int>(static_cast<uint32_t>(v >> 32)));
  return (static_cast<uint64_t>(static_cast<uint32_t>(hi)) << 32) | static_cast<uint32_t>(lo);
}

template <int G>
__device__ __forceinline__ uint64_t group_max64(uint64_t v) {
  if constexpr (G > 1) v = umax64(v, dpp_u64<kDppSwap1>(v));
  if constexpr (G > 2) v = umax64(v, dpp_u64<kDppSwap2>(v));
  if constexpr (G > 4) v = umax64(v, dpp_u64<kDppHalfMirror>(v));
  if constexpr (G > 8) v = umax64(v, dpp_u64<kDppMirror>(v));
  if constexpr (G > 16) v = umax64(v, __shfl_xor(static_cast<unsigned long long>(v), 16));
  if constexpr (G > 32) v = umax64(v, __shfl_xor(static_cast<unsigned long long>(v), 32));
  return v;
}

template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
  return __int_as_float(dpp_i32<CTRL>(__float_as_int(v)));
}

// Each level adds the same two partial sums on both lanes of a pair, so every
// lane of the group ends with the same bits.
template <int G>
__device__ __forceinline__ float group_sum(float v) {
  if constexpr (G > 1) v += dpp_f32<kDppSwap1>(v);
  if constexpr (G > 2) v += dpp_f32<kDppSwap2>(v);
  if constexpr (G > 4) v += dpp_f32<kDppHalfMirror>(v);
  if constexpr (G > 8) v += dpp_f32<kDppMirror>(v);
  if constexpr (G > 16) v += __shfl_xor(v, 16);
  if constexpr (G > 32) v += __shfl_xor(v, 32);
  return v;
}

template <int G, int V, bool EXT>
__global__ __launch_bounds__(kBlock) void route_kernel(RouteKernelArgs a) {
  extern __shared__ int hist[];
  constexpr int kGroups = kBlock / G;
  const int T = a.T, E = a.E, k = a.k;
  const bool stats = a.counts != nullptr;
  const bool use_lds = a.lds_bins > 0;
  const int tid = threadIdx.x;
  const int gl = tid & (G - 1);
  const int group = tid / G;
  // group-limit staging: one row of E selection values per token group,
  // after the histogram
  float* cval = reinterpret_cast<float*>(hist + a.lds_bins) + group * E;
  const bool grouped = EXT && a.n_group > 1;
  const int gsz = grouped ? E / a.n_group : E;
  // one block routing the whole batch also dispatches it: the dispatch's
  // tables, then the pairs' expert ids (T k ints)
  int* disp_sm = hist + a.lds_bins + (grouped ? kGroups * E : 0);
  int* disp_ids = disp_sm + dispatch_one_block_ints(E, a.d.E_local);
  if (stats && use_lds) {
    for (int b = tid; b < a.lds_bins; b += kBlock) hist[b] = 0;
    __syncthreads();
  }
  const int t0 = blockIdx.x * a.tokens_per_block;
  const int t1 = min(T, t0 + a.tokens_per_block);
  // The loads of a token group's pass: all V logits (and its source) go out
  // before the first is used, and those of the block's next pass (a block
  // that routes the whole batch makes up to four) go out before this pass
  // computes.  A lane past the row or the batch reads element 0 (T >= 1)
  // and discards it, so no load sits in a branch of its own behind the
  // previous one's wait.
  const bool biased = EXT && a.gate == 2 && a.bias != nullptr;
  float braw[V];
#pragma unroll
  for (int v = 0; v < V; ++v) {
    const int e = gl + G * v;
    braw[v] = biased ? a.bias[e < E ? e : 0] : 0.0f;
  }
  float nraw[V];
  int nsrc = 0;
  auto load_pass = [&](int b) {
    const int tt = b + group;
    const bool ok = tt < t1;
    nsrc = stats ? a.src[ok ? tt : 0] : 0;
#pragma unroll
    for (int v = 0; v < V; ++v) {
      const int e = gl + G * v;
      nraw[v] = a.logits[(ok && e < E) ? static_cast<size_t>(tt) * E + e : 0];
    }
  };
  if (t0 < t1) load_pass(t0);
  for (int base = t0; base < t1; base += kGroups) {
    const int t = base + group;
    const bool valid = t < t1;
    uint64_t key[V];
    float lg[V];
    float raw[V];
#pragma unroll
    for (int v = 0; v < V; ++v) raw[v] = nraw[v];
    const int src_t = nsrc;
    if (base + kGroups < t1) load_pass(base + kGroups);
#pragma unroll
    for (int v = 0; v < V; ++v) {
      const int e = gl + G * v;
      key[v] = 0;
      lg[v] = __builtin_nanf("");
      if (valid && e < E) {
        const float f = raw[v];
        lg[v] = f;
        float c = f;
        if (EXT && a.gate == 2) {
          c = sigmoid_score(f);
          if (biased) c = c + braw[v];
        }
        if (grouped) cval[e] = c;
        key[v] = (static_cast<uint64_t>(order_key(c)) << 32) | static_cast<uint32_t>(~e);
      }
    }
    if (grouped) {
      // the group's lanes share this wave: a block-wide barrier is not needed
      // between its LDS writes and reads, only the LDS wait
      __builtin_amdgcn_s_waitcnt(0xc07f);
      __builtin_amdgcn_wave_barrier();
      // the two first selection values of each expert group, then their sum:
      // L lanes per group (L = G / n_group when that divides the group
      // evenly, else 1), lane j of group q scanning elements j, j + L, ...,
      // and the lanes' top-2 pairs merged by exchanges within the L lanes
      const int L = (G % a.n_group == 0 && gsz % (G / a.n_group) == 0) ? G / a.n_group : 1;
      const int q_mine = gl / L, j_mine = gl % L;
      uint64_t k1 = 0, k2 = 0;
      if (valid && q_mine < a.n_group) {
        for (int i = j_mine; i < gsz; i += L) {
          const int e = q_mine * gsz + i;
          const uint64_t ke = (static_cast<uint64_t>(order_key(cval[e])) << 32) | static_cast<uint32_t>(~e);
          if (ke > k1) {
            k2 = k1;
            k1 = ke;
          } else if (ke > k2) {
            k2 = ke;
          }
        }
      }
      for (int off = 1; off < L; off <<= 1) {
        const uint64_t o1 = __shfl_xor(static_cast<unsigned long long>(k1), off);
        const uint64_t o2 = __shfl_xor(static_cast<unsigned long long>(k2), off);
        // top two of {k1, k2, o1, o2}; keys are distinct (the expert id is in them) or 0
        const uint64_t hi = umax64(k1, o1), lo = k1 > o1 ? o1 : k1;
        k2 = umax64(lo, umax64(k2, o2));
        k1 = hi;
      }
      uint64_t gkey = 0;   // every lane of group q holds the group's key
      if (valid && q_mine < a.n_group) {
        const float c1 = cval[~static_cast<uint32_t>(k1)];
        const float gs = gsz > 1 ? c1 + cval[~static_cast<uint32_t>(k2)] : c1;
        gkey = (static_cast<uint64_t>(order_key(gs)) << 32) | static_cast<uint32_t>(~q_mine);
      }
      uint64_t kept = 0;   // bit q: group q stays
      for (int r = 0; r < a.topk_group; ++r) {
        const uint64_t best = group_max64<G>(gkey);
        if (best == 0) break;   // a token group past the batch end
        const int q = static_cast<int>(~static_cast<uint32_t>(best));
        kept |= 1ull << q;
        if (q_mine == q) gkey = 0;
      }
#pragma unroll
      for (int v = 0; v < V; ++v) {
        const int e = gl + G * v;
        if (e < E && !((kept >> (e / gsz)) & 1ull)) key[v] = 0;
      }
      // the next token's writes must not overtake this token's reads
      __builtin_amdgcn_s_waitcnt(0xc07f);
      __builtin_amdgcn_wave_barrier();
    }
    uint32_t my_key = 0;
    int my_e = 0;
    for (int r = 0; r < k; ++r) {
      uint64_t best = key[0];
#pragma unroll
      for (int v = 1; v < V; ++v) best = umax64(best, key[v]);
      best = group_max64<G>(best);
      const int e = static_cast<int>(~static_cast<uint32_t>(best));
#pragma unroll
      for (int v = 0; v < V; ++v)
        if (e == gl + G * v) key[v] = 0;
      if (gl == r) {
        my_key = static_cast<uint32_t>(best >> 32);
        my_e = e;
      }
    }
    float wgt;
    if (!EXT || a.gate == 0) {
      const float val = key_value(my_key);
      const float m = __shfl(val, 0, G);
      const float ex = (gl < k) ? expf(val - m) : 0.0f;
      wgt = ex / group_sum<G>(ex);
    } else if (a.gate == 1) {
      // softmax over all E logits: M is the largest logit that is a number,
      // then every exp(l - M) is summed
      uint32_t mk = 0;
#pragma unroll
      for (int v = 0; v < V; ++v)
        if (lg[v] == lg[v]) mk = max(mk, order_key(lg[v]));
      mk = static_cast<uint32_t>(group_max64<G>(mk) & 0xffffffffu);
      const float M = mk ? key_value(mk) : __builtin_nanf("");
      float part = 0.0f;
#pragma unroll
      for (int v = 0; v < V; ++v)
        if (gl + G * v < E) part += expf(lg[v] - M);
      const float sum = group_sum<G>(part);
      const float lj = (valid && gl < k) ? a.logits[static_cast<size_t>(t) * E + my_e] : 0.0f;
      wgt = expf(lj - M) / sum;
    } else {
      // picked sigmoid scores renormalised over the picks
      const float sj = (valid && gl < k) ? sigmoid_score(a.logits[static_cast<size_t>(t) * E + my_e]) : 0.0f;
      wgt = sj / group_sum<G>(sj);
    }
    if (EXT) wgt *= a.scale;
    if (valid && gl < k) {
      const size_t o = static_cast<size_t>(t) * k + gl;
      a.topk_idx[o] = my_e;
      a.topk_w[o] = wgt;
      if (a.disp) disp_ids[o] = my_e;   // (o < kDispatchPairs: one block routes the batch)
      if (stats) count_pair(src_t, my_e, a.S, E, use_lds, hist, a.counts, a.expert_load);
    }
  }
  if (stats && use_lds) {
    __syncthreads();
    flush_hist(hist, a.lds_bins, E, a.counts, a.expert_load);
  }
  if (a.disp) {
    // this block routed the whole batch: its expert ids are in disp_ids
    __syncthreads();
    dispatch_one_block(T * k, k, E, a.d.E_local, a.d.local_experts, disp_ids, a.d.offsets, a.d.perm_token,
                       a.d.inv_pos, disp_sm);
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

template <int G, int V, bool EXT>
hipError_t launch_route_gv(const RouteKernelArgs& in, hipStream_t st, bool* dispatched) {
  constexpr int kGroups = kBlock / G;
  RouteKernelArgs a = in;
  // One token per group and block: the selection is a chain of dependent
  // lane reductions, so many resident blocks hide its latency.  A batch
  // whose dispatch fits one block (at most kDispatchPairs pairs, four token
  // groups) is routed by a single block that then also dispatches it,
  // which saves a launch for decode-sized batches.
  a.tokens_per_block = kGroups;
  if (a.disp && (static_cast<long long>(a.T) * a.k > kDispatchPairs || a.T > 4 * kGroups || a.d.E_local > kBlock))
    a.disp = false;
  if (a.disp) a.tokens_per_block = a.T;
  a.lds_bins = (a.counts && a.S * a.E <= kLdsBinsMax) ? a.S * a.E : 0;
  const int blocks = ceil_div(a.T, a.tokens_per_block);
  // histogram (at most 64 KB), group-limit staging (EXT), dispatch tables
  // and expert ids;
  // the block-scan's partial sums take 64 more bytes of static LDS
  const size_t lds = a.lds_bins * sizeof(int) + ((EXT && a.n_group > 1) ? sizeof(float) * kGroups * a.E : 0) +
                     (a.disp ? sizeof(int) * (dispatch_one_block_ints(a.E, a.d.E_local) + kDispatchPairs) : 0);
  if (dispatched) *dispatched = a.disp;
  static unsigned long long lds_set = 0;  // devices with the LDS limit raised
  const hipError_t e_lds =
      set_max_dynamic_lds(reinterpret_cast<const void*>(&route_kernel<G, V, EXT>), 160 * 1024 - 1024, &lds_set);
  if (e_lds != hipSuccess) return e_lds;
  hipLaunchKernelGGL((route_kernel<G, V, EXT>), dim3(blocks), dim3(kBlock), lds, st, a);
  return hipGetLastError();
}

template <int G, bool EXT>
hipError_t launch_route_g(const RouteKernelArgs& a, int V, hipStream_t st, bool* dispatched) {
  switch (V) {
    case 1: return launch_route_gv<G, 1, EXT>(a, st, dispatched);
    case 2: return launch_route_gv<G, 2, EXT>(a, st, dispatched);
    case 4: return launch_route_gv<G, 4, EXT>(a, st, dispatched);
    case 8: return launch_route_gv<G, 8, EXT>(a, st, dispatched);
    default: return launch_route_gv<G, 16, EXT>(a, st, dispatched);
  }
}

// Lanes per token G and logits per lane V: G covers E when E <= 16;
// otherwise the narrowest G >= 16 that holds the picks (k) and the expert
// groups (one lane each), with at most 16 logits per lane (8 for the gating
// variants) below 1024 experts.  Narrow groups route more tokens per wave
// (half the waves: the whole grid of a 16384-token batch resident at once),
// and a max over 16 lanes is four DPP steps within a row.
template <bool EXT>
hipError_t launch_route_ext(const RouteKernelArgs& a, hipStream_t st, bool* dispatched) {
  const int E = a.E;
  const int need = max(a.k, EXT && a.n_group > 1 ? a.n_group : 1);
  int G = 2;
  if (E <= 16) {
    while (G < E) G *= 2;
  } else {
    // at most 16 logits per lane (8 with the gating variants, whose extra
    // state would otherwise halve the resident waves)
    const int v_max = EXT ? 8 : 16;
    G = 16;
    while (G < 64 && (G < need || E > v_max * G)) G *= 2;
  }
  int V = 1;
  while (V * G < E) V *= 2;
  switch (G) {
    case 2: return launch_route_g<2, EXT>(a, V, st, dispatched);
    case 4: return launch_route_g<4, EXT>(a, V, st, dispatched);
    case 8: return launch_route_g<8, EXT>(a, V, st, dispatched);
    case 16: return launch_route_g<16, EXT>(a, V, st, dispatched);
    case 32: return launch_route_g<32, EXT>(a, V, st, dispatched);
    default: return launch_route_g<64, EXT>(a, V, st, dispatched);
  }
}

}  // namespace

hipError_t launch_route(int T, int E, int k, const float* logits, int32_t* topk_idx,
                        float* topk_w, const int32_t* src, int S, int64_t* counts,
                        int32_t* expert_load, const RouteGating* gating, hipStream_t st,
                        const DispatchArgs* dispatch, bool* dispatched) {
  if (dispatched) *dispatched = false;
  if (T == 0) return hipSuccess;
  RouteKernelArgs a{};
  if (dispatch) {
    a.disp = true;
    a.d = *dispatch;
  }
  a.T = T;
  a.E = E;
  a.k = k;
  a.logits = logits;
  a.topk_idx = topk_idx;
  a.topk_w = topk_w;
  a.src = src;
  a.S = S;
  a.counts = reinterpret_cast<unsigned long long*>(counts);
  a.expert_load = expert_load;
  a.scale = 1.0f;
  const bool ext = gating && (gating->gate != 0 || gating->bias || gating->n_group > 1 || gating->scale != 1.0f);
  if (ext) {
    a.gate = gating->gate;
    a.bias = gating->bias;
    a.scale = gating->scale;
    a.n_group = gating->n_group;
    a.topk_group = gating->topk_group;
  }
  return ext ? launch_route_ext<true>(a, st, dispatched) : launch_route_ext<false>(a, st, dispatched);
}

hipError_t launch_route_stats(int T, int k, int S, int E, const int32_t* src,
                              const int32_t* topk_idx, int64_t* counts, int32_t* expert_load,
                              hipStream_t st) {
  const int n_pairs = T * k;
  if (n_pairs == 0) return hipSuccess;
  const int pairs_per_block = kStatsPairs;
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
