// Source-aware expert placement on the GPU: the online greedy of Sec. 5.3
// over the objective of Sec. 5.2, one workgroup per MoE layer.
//
// The statistics it consumes (the source x expert matrix A and the aggregate
// load B, Sec. 5.1) are accumulated on the device by the routing kernels, so
// the placement runs where they already are.  Per layer:
//   1. every thread sums the source-aware volume V_e = sum_s A_{s,e} of its
//      experts and stages B, V, the current ranks x^0 and the source/rank cost
//      matrix D in LDS;
//   2. every thread ranks its experts by hotness (B descending, then V
//      descending, then lower index) by counting the experts ahead of them;
//   3. hottest first, in chunks: all waves compute the chunk's placement-
//      independent terms C^comm = sum_s A_{s,e} D_{s,g} and C^mig (zero on
//      the current rank, else M_{e,g} plus M_{e,x0} when x0 is a rank) into
//      LDS; then wave 0 places the chunk's experts one at a time, lane g
//      scoring rank g with the load term C^load = (L_g + B_e - Lbar)^2 -
//      (L_g - Lbar)^2 that depends on the experts placed before, and a
//      butterfly over the lanes picks the lowest score (ties: the current
//      rank, then fewer experts placed, then the lower rank);
//   4. the placement, each rank's experts and the objective's three terms of
//      the result are written out.
// Scores are fp64 and evaluated left to right without contraction into fused
// multiply-adds, so the chosen rank is the one any IEEE fp64 evaluation of the
// same expressions chooses.
#include "common.h"
#include "kernels.h"

#pragma clang fp contract(off)

namespace moe {
namespace {

constexpr int kPlaceThreads = 256;
constexpr int kPlaceWaves = kPlaceThreads / kWave;

struct PlaceKernelArgs {
  const int64_t* A;
  const int64_t* B;
  const double* D;
  const double* M;
  const int32_t* x0;
  int32_t* x;
  int32_t* rank_experts;
  double* cost;
  double alpha, beta, gamma, m_uniform;
  int S, E, G, slots, chunk;
  int cap[kPlaceMaxRanks];
};

typedef int64_t i64x2 __attribute__((ext_vector_type(2)));

struct PlaceLds {
  i64x2* bv;       // [E] (B, V) of each expert: aggregate load, source-aware volume
  double* D;       // [S*G]
  double2* terms;  // [chunk*G] (C^comm, C^mig) of the staged chunk
  int64_t* bo;     // [E] B of the expert in hotness position i
  int32_t* order;  // [E] expert in hotness position i
  int32_t* ho;     // [E] x^0 of the expert in hotness position i
  int32_t* xpos;   // [E] rank chosen for hotness position i
  int32_t* xs;     // [E] rank chosen for each expert
  int32_t* fill;   // [kPlaceMaxRanks] experts placed per rank
  int64_t* red_i;  // [2 * kPlaceWaves]
  double* red_d;   // [2 * kPlaceWaves]
  int64_t* A;      // [S*E] this layer's counts when they fit (a_staged), else
                   // [chunk][S] the columns of the staged chunk's experts
};

// The layer's A is staged in LDS when it takes at most this many bytes;
// otherwise each chunk stages its experts' columns, at most as many bytes.
constexpr size_t kStageABytes = 32 * 1024;
__host__ __device__ inline bool a_staged(int S, int E) {
  return static_cast<size_t>(S) * E * sizeof(int64_t) <= kStageABytes;
}

// Experts per staged chunk: at most 2048 (expert, rank) terms, and when A is
// not staged whole, at most kStageABytes of A columns.
__host__ __device__ inline int place_chunk_experts(int S, int E, int G) {
  int c = 2048 / G;
  if (!a_staged(S, E)) c = c < static_cast<int>(kStageABytes / (8 * S)) ? c : static_cast<int>(kStageABytes / (8 * S));
  c = c < E ? c : E;
  return c > 1 ? c : 1;
}

__host__ __device__ inline size_t align16(size_t v) { return (v + 15) & ~static_cast<size_t>(15); }

// Byte offsets of the LDS carve; the same function sizes the launch.
__host__ __device__ inline size_t place_lds_layout(int S, int E, int G, int chunk, size_t* off) {
  size_t o = 0;
  off[0] = o; o = align16(o + 16 * static_cast<size_t>(E));                 // bv
  off[1] = o; o = align16(o + sizeof(double) * S * G);                      // D
  off[2] = o; o = align16(o + sizeof(double2) * chunk * G);                 // terms
  off[3] = o; o = align16(o + sizeof(int64_t) * E);                         // bo
  off[4] = o; o = align16(o + sizeof(int32_t) * E);                         // order
  off[5] = o; o = align16(o + sizeof(int32_t) * E);                         // ho
  off[6] = o; o = align16(o + sizeof(int32_t) * E);                         // xpos
  off[7] = o; o = align16(o + sizeof(int32_t) * E);                         // xs
  off[8] = o; o = align16(o + sizeof(int32_t) * kPlaceMaxRanks);            // fill
  off[9] = o; o = align16(o + sizeof(int64_t) * 2 * kPlaceWaves);           // red_i
  off[10] = o; o = align16(o + sizeof(double) * 2 * kPlaceWaves);           // red_d
  off[11] = o;
  o = align16(o + sizeof(int64_t) * S * (a_staged(S, E) ? E : chunk));       // A or its columns
  return o;
}
constexpr int kLdsParts = 12;

__device__ __forceinline__ double mig_cost(const PlaceKernelArgs& a, int l, int e, int g) {
  return a.M ? a.M[(static_cast<size_t>(l) * a.E + e) * a.G + g] : a.m_uniform;
}

// C^mig of expert e on rank g: zero on its current rank, else the two
// indicator changes M_{e,g} and (when it has a rank) M_{e,home}.
__device__ __forceinline__ double mig_term(const PlaceKernelArgs& a, int l, int e, int g, int home) {
  const bool home_ok = home >= 0 && home < a.G;
  if (home_ok && g == home) return 0.0;
  double m = mig_cost(a, l, e, g);
  if (home_ok) m = m + mig_cost(a, l, e, home);
  return m;
}

// C^comm of an expert on rank g: sum_s A_{s,e} D_{s,g}, in s order, with
// A_{s,e} = col[s * stride] (the layer's A in LDS, or its staged column);
// eight loads are issued before their products are summed.
__device__ __forceinline__ double comm_term(const int64_t* col, int stride, const double* D, int S, int G,
                                            int g) {
  double comm = 0.0;
  int src = 0;
  for (; src + 8 <= S; src += 8) {
    int64_t av[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) av[j] = col[(src + j) * stride];
#pragma unroll
    for (int j = 0; j < 8; ++j) comm = comm + static_cast<double>(av[j]) * D[(src + j) * G + g];
  }
  for (; src < S; ++src) comm = comm + static_cast<double>(col[src * stride]) * D[src * G + g];
  return comm;
}

template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t v) {
  return static_cast<uint32_t>(
      __builtin_amdgcn_update_dpp(static_cast<int>(v), static_cast<int>(v), CTRL, 0xf, 0xf, false));
}
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double v) {
  const int lo = __builtin_amdgcn_update_dpp(__double2loint(v), __double2loint(v), CTRL, 0xf, 0xf, false);
  const int hi = __builtin_amdgcn_update_dpp(__double2hiint(v), __double2hiint(v), CTRL, 0xf, 0xf, false);
  return __hiloint2double(hi, lo);
}
// Scores are never NaN here (a NaN score is replaced by +inf first), so the
// hardware minimum is exact; of -0.0 and +0.0 it may return either, which the
// equality test of the tie phase treats alike.
__device__ __forceinline__ double min_f64(double a, double b) { return __builtin_fmin(a, b); }
__device__ __forceinline__ uint32_t min_u32(uint32_t a, uint32_t b) { return b < a ? b : a; }

// DPP controls: swap neighbours, swap pairs, mirror each half row (lane i <->
// 7 - i), mirror each row (lane i <-> 15 - i).  After the four levels every
// lane of a 16-lane row holds the row's minimum.
constexpr int kDppSwap1 = 0xB1;   // quad_perm [1, 0, 3, 2]
constexpr int kDppSwap2 = 0x4E;   // quad_perm [2, 3, 0, 1]
constexpr int kDppHalfMirror = 0x141;
constexpr int kDppMirror = 0x140;

// Minimum over the first 2^LEVELS lanes (every lane among them gets it;
// lanes past G must hold values that do not win).
template <int LEVELS>
__device__ __forceinline__ double lanes_min_f64(double v) {
  if constexpr (LEVELS > 0) v = min_f64(v, dpp_f64<kDppSwap1>(v));
  if constexpr (LEVELS > 1) v = min_f64(v, dpp_f64<kDppSwap2>(v));
  if constexpr (LEVELS > 2) v = min_f64(v, dpp_f64<kDppHalfMirror>(v));
  if constexpr (LEVELS > 3) v = min_f64(v, dpp_f64<kDppMirror>(v));
  if constexpr (LEVELS > 4) v = min_f64(v, __shfl_xor(v, 16));
  if constexpr (LEVELS > 5) v = min_f64(v, __shfl_xor(v, 32));
  return v;
}
template <int LEVELS>
__device__ __forceinline__ uint32_t lanes_min_u32(uint32_t v) {
  if constexpr (LEVELS > 0) v = min_u32(v, dpp_u32<kDppSwap1>(v));
  if constexpr (LEVELS > 1) v = min_u32(v, dpp_u32<kDppSwap2>(v));
  if constexpr (LEVELS > 2) v = min_u32(v, dpp_u32<kDppHalfMirror>(v));
  if constexpr (LEVELS > 3) v = min_u32(v, dpp_u32<kDppMirror>(v));
  if constexpr (LEVELS > 4) v = min_u32(v, __shfl_xor(v, 16));
  if constexpr (LEVELS > 5) v = min_u32(v, __shfl_xor(v, 32));
  return v;
}

// State of rank g, held by lane g of wave 0: experts placed, load placed (as
// int64, and as an exact double in FAST mode), u2 = (L_g - Lbar)^2, and the
// C^comm and C^mig of the experts it won.
struct RankState {
  int placed;
  int64_t load;
  double loadd, u2, comm, mig;
};

// Wave 0's greedy over one staged chunk of nc hotness positions from c0.
// FAST requires every partial load to be an integer below 2^53, so that
// (double)(L + B) equals the double sum of the two exact conversions.
template <bool FAST, int LEVELS>
__device__ __forceinline__ void place_chunk_steps(const PlaceKernelArgs& a, const PlaceLds& s, int c0, int nc,
                                                  double mean, int lane, int cap_g, RankState& r) {
  const int G = a.G;
  const int gl = lane < G ? lane : G - 1;   // lanes past G read a valid term and stay closed
  double2 t_next = s.terms[gl];
  int64_t be_next = s.bo[c0];
  int home_next = s.ho[c0];
  int xw = 0;   // lane j keeps the rank of step j of the current 64
  for (int i = 0; i < nc; ++i) {
    const double2 t = t_next;
    const int64_t be = be_next;
    const int home = home_next;
    const int in = min(i + 1, nc - 1);
    t_next = s.terms[in * G + gl];
    be_next = s.bo[c0 + in];
    home_next = s.ho[c0 + in];

    const bool open = r.placed < cap_g;
    const double bd = static_cast<double>(be);
    const double v = (FAST ? r.loadd + bd : static_cast<double>(r.load + be)) - mean;
    const double vv = v * v;
    const double c_load = vv - r.u2;
    double score = a.alpha * t.x;
    score = score + a.beta * c_load;
    score = score + a.gamma * t.y;
    score = (open & (score == score)) ? score : __builtin_inf();
    // ties: a full rank loses, then the current rank wins, then fewer
    // experts placed, then the lower rank
    const uint32_t key = (open ? 0u : 0x80000000u) | (lane == home ? 0u : 0x40000000u) |
                         (static_cast<uint32_t>(r.placed) << 6) | static_cast<uint32_t>(lane);
    const double best = lanes_min_f64<LEVELS>(score);
    const uint32_t k = lanes_min_u32<LEVELS>(score == best ? key : 0xffffffffu);
    const int w = static_cast<int>(__builtin_amdgcn_readfirstlane(k) & 63u);
    const bool won = lane == w;
    r.placed += won ? 1 : 0;
    if (FAST)
      r.loadd = won ? r.loadd + bd : r.loadd;
    else
      r.load += won ? be : 0;
    r.u2 = won ? vv : r.u2;   // the new load's (L - Lbar) is this step's v
    r.comm = won ? r.comm + t.x : r.comm;
    r.mig = won ? r.mig + t.y : r.mig;
    xw = lane == (i & 63) ? w : xw;
    if ((i & 63) == 63 || i == nc - 1) {
      if (lane <= (i & 63)) s.xpos[c0 + (i & ~63) + lane] = xw;
    }
  }
}

__device__ __forceinline__ int64_t wave_sum_i64(int64_t v) {
  for (int off = kWave / 2; off > 0; off >>= 1) v += __shfl_xor(v, off);
  return v;
}

__device__ __forceinline__ double wave_sum_f64(double v) {
  for (int off = kWave / 2; off > 0; off >>= 1) v = v + __shfl_xor(v, off);
  return v;
}

__global__ __launch_bounds__(kPlaceThreads) void place_kernel(PlaceKernelArgs a) {
  extern __shared__ __align__(16) unsigned char place_smem[];
  const int l = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int S = a.S, E = a.E, G = a.G;
  const int64_t* A_l = a.A + static_cast<size_t>(l) * S * E;
  const int32_t* x0_l = a.x0 + static_cast<size_t>(l) * E;

  size_t off[kLdsParts];
  place_lds_layout(S, E, G, a.chunk, off);
  PlaceLds s;
  s.bv = reinterpret_cast<i64x2*>(place_smem + off[0]);
  s.D = reinterpret_cast<double*>(place_smem + off[1]);
  s.terms = reinterpret_cast<double2*>(place_smem + off[2]);
  s.bo = reinterpret_cast<int64_t*>(place_smem + off[3]);
  s.order = reinterpret_cast<int32_t*>(place_smem + off[4]);
  s.ho = reinterpret_cast<int32_t*>(place_smem + off[5]);
  s.xpos = reinterpret_cast<int32_t*>(place_smem + off[6]);
  s.xs = reinterpret_cast<int32_t*>(place_smem + off[7]);
  s.fill = reinterpret_cast<int32_t*>(place_smem + off[8]);
  s.red_i = reinterpret_cast<int64_t*>(place_smem + off[9]);
  s.red_d = reinterpret_cast<double*>(place_smem + off[10]);
  const bool staged = a_staged(S, E);
  s.A = reinterpret_cast<int64_t*>(place_smem + off[11]);

  // 1. hotness signals, D, and the layer's A when it fits in LDS
  int64_t part = 0;
  int negative = 0;
  for (int e = tid; e < E; e += kPlaceThreads) {
    int64_t v = 0;
#pragma unroll 8
    for (int src = 0; src < S; ++src) {
      const int64_t c = A_l[static_cast<size_t>(src) * E + e];
      if (staged) s.A[src * E + e] = c;
      v += c;
    }
    const int64_t b = a.B ? a.B[static_cast<size_t>(l) * E + e] : v;
    i64x2 bv;
    bv.x = b;
    bv.y = v;
    s.bv[e] = bv;
    part += b;
    negative |= static_cast<int>(b < 0);
  }
  for (int i = tid; i < S * G; i += kPlaceThreads) s.D[i] = a.D[i];
  part = wave_sum_i64(part);
  const int64_t neg_w = wave_sum_i64(negative);
  if (lane == 0) {
    s.red_i[wave] = part;
    s.red_i[kPlaceWaves + wave] = neg_w;
  }
  __syncthreads();
  int64_t total = 0, n_negative = 0;
  for (int w = 0; w < kPlaceWaves; ++w) {
    total += s.red_i[w];
    n_negative += s.red_i[kPlaceWaves + w];
  }
  // every expert is placed, so the final average rank load is known up front
  const double mean = static_cast<double>(total) / G;
  // non-negative loads whose total is below 2^53: every partial load is an
  // exactly representable integer
  const bool fast = n_negative == 0 && total < (int64_t{1} << 53);

  // 2. hotness order: an expert's position is the number of experts ahead of
  // it; tpe consecutive lanes split the count of one expert
  int tpe = 1;
  while (tpe < kWave && tpe * 2 * E <= kPlaceThreads) tpe *= 2;
  for (int idx = tid; idx < E * tpe; idx += kPlaceThreads) {
    const int e = idx / tpe;
    const int sub = idx - e * tpe;
    const i64x2 me = s.bv[e];
    auto before = [&](const i64x2 o, int f) {
      return static_cast<int>((o.x > me.x) | ((o.x == me.x) & ((o.y > me.y) | ((o.y == me.y) & (f < e)))));
    };
    int ahead = 0;
    int f = sub;
    for (; f + 3 * tpe < E; f += 4 * tpe) {   // four independent loads per round
      const i64x2 o0 = s.bv[f], o1 = s.bv[f + tpe], o2 = s.bv[f + 2 * tpe], o3 = s.bv[f + 3 * tpe];
      ahead += before(o0, f) + before(o1, f + tpe) + before(o2, f + 2 * tpe) + before(o3, f + 3 * tpe);
    }
    for (; f < E; f += tpe) ahead += before(s.bv[f], f);
    for (int m = tpe / 2; m > 0; m >>= 1) ahead += __shfl_xor(ahead, m);
    if (sub == 0) {
      s.order[ahead] = e;
      s.bo[ahead] = me.x;
      s.ho[ahead] = x0_l[e];
    }
  }
  __syncthreads();

  // 3. greedy, hottest first; wave 0 lane g keeps rank g's state
  RankState r{0, 0, 0.0, mean * mean, 0.0, 0.0};   // u2 = (0 - mean)^2
  const int cap_g = lane < G ? a.cap[lane] : 0;
  int levels = 0;   // butterfly levels that cover G lanes
  while ((1 << levels) < G) ++levels;
  for (int c0 = 0; c0 < E; c0 += a.chunk) {
    const int nc = min(a.chunk, E - c0);
    if (!staged) {   // this chunk's columns of A, [i][S]
      for (int q = tid; q < nc * S; q += kPlaceThreads) {
        const int i = q / S;
        const int src = q - i * S;
        s.A[q] = A_l[static_cast<size_t>(src) * E + s.order[c0 + i]];
      }
      __syncthreads();
    }
    for (int p = tid; p < nc * G; p += kPlaceThreads) {
      const int i = p / G;
      const int g = p - i * G;
      const int e = s.order[c0 + i];
      const double comm = staged ? comm_term(s.A + e, E, s.D, S, G, g) : comm_term(s.A + i * S, 1, s.D, S, G, g);
      const double mig = mig_term(a, l, e, g, s.ho[c0 + i]);
      s.terms[p] = make_double2(comm, mig);
    }
    __syncthreads();
    if (wave == 0) {
      switch ((fast ? 8 : 0) + levels) {
#define PLACE_STEPS(F, LV)                                              \
  case (F ? 8 : 0) + LV:                                                \
    place_chunk_steps<F, LV>(a, s, c0, nc, mean, lane, cap_g, r);      \
    break;
        PLACE_STEPS(true, 0) PLACE_STEPS(true, 1) PLACE_STEPS(true, 2) PLACE_STEPS(true, 3)
        PLACE_STEPS(true, 4) PLACE_STEPS(true, 5) PLACE_STEPS(true, 6)
        PLACE_STEPS(false, 0) PLACE_STEPS(false, 1) PLACE_STEPS(false, 2) PLACE_STEPS(false, 3)
        PLACE_STEPS(false, 4) PLACE_STEPS(false, 5) PLACE_STEPS(false, 6)
#undef PLACE_STEPS
        default: break;
      }
    }
    __syncthreads();
  }

  // 4. results: the objective's terms from the ranks' sums, the placement by
  // expert, and each rank's experts in ascending order
  for (int i = tid; i < E; i += kPlaceThreads) s.xs[s.order[i]] = s.xpos[i];
  if (wave == 0) {
    if (lane < G) s.fill[lane] = r.placed;
    if (a.cost) {
      const bool rank = lane < G;
      const double c_comm = wave_sum_f64(rank ? r.comm : 0.0);
      const double c_load = wave_sum_f64(rank ? r.u2 : 0.0);
      const double c_mig = wave_sum_f64(rank ? r.mig : 0.0);
      if (lane == 0) {
        a.cost[static_cast<size_t>(l) * 3 + 0] = c_comm;
        a.cost[static_cast<size_t>(l) * 3 + 1] = c_load;
        a.cost[static_cast<size_t>(l) * 3 + 2] = c_mig;
      }
    }
  }
  __syncthreads();
  for (int e = tid; e < E; e += kPlaceThreads) {
    const int g = s.xs[e];
    a.x[static_cast<size_t>(l) * E + e] = g;
    if (a.rank_experts) {
      int pos = 0;
      for (int f = 0; f < e; ++f) pos += static_cast<int>(s.xs[f] == g);
      a.rank_experts[(static_cast<size_t>(l) * G + g) * a.slots + pos] = e;
    }
  }
  if (a.rank_experts) {
    for (int i = tid; i < G * a.slots; i += kPlaceThreads) {
      const int g = i / a.slots;
      if (i - g * a.slots >= s.fill[g])
        a.rank_experts[static_cast<size_t>(l) * G * a.slots + i] = -1;
    }
  }
}

}  // namespace

size_t place_lds_bytes(int S, int E, int G) {
  size_t off[kLdsParts];
  return place_lds_layout(S, E, G, place_chunk_experts(S, E, G), off);
}

hipError_t launch_place(const PlaceArgs& h, hipStream_t st) {
  if (h.L == 0) return hipSuccess;
  PlaceKernelArgs a{};
  a.A = h.A;
  a.B = h.B;
  a.D = h.D;
  a.M = h.M;
  a.x0 = h.x0;
  a.x = h.x;
  a.rank_experts = h.rank_experts;
  a.cost = h.cost;
  a.alpha = h.alpha;
  a.beta = h.beta;
  a.gamma = h.gamma;
  a.m_uniform = h.m_uniform;
  a.S = h.S;
  a.E = h.E;
  a.G = h.G;
  a.slots = h.slots;
  a.chunk = place_chunk_experts(h.S, h.E, h.G);
  for (int g = 0; g < h.G; ++g) a.cap[g] = h.cap[g];
  const size_t lds = place_lds_bytes(h.S, h.E, h.G);
  static unsigned long long lds_set = 0;  // devices with the LDS limit raised
  const hipError_t e_lds =
      set_max_dynamic_lds(reinterpret_cast<const void*>(&place_kernel),
                          kPlaceMaxLdsBytes, &lds_set);
  if (e_lds != hipSuccess) return e_lds;
  hipLaunchKernelGGL(place_kernel, dim3(h.L), dim3(kPlaceThreads), lds, st, a);
  return hipGetLastError();
}

}  // namespace moe
