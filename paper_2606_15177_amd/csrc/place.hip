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
constexpr int kChunkTerms = 2048;  // (expert, rank) term pairs staged per chunk

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

struct PlaceLds {
  int64_t* B;      // [E] aggregate load
  int64_t* V;      // [E] source-aware volume
  double* D;       // [S*G]
  double2* terms;  // [chunk*G] (C^comm, C^mig) of the staged chunk
  double2* won;    // [E] (C^comm, C^mig) at the chosen rank
  int64_t* bo;     // [E] B of the expert in hotness position i
  int32_t* order;  // [E] expert in hotness position i
  int32_t* home;   // [E] x^0 by expert
  int32_t* xs;     // [E] chosen rank by expert
  int32_t* fill;   // [kPlaceMaxRanks] experts placed per rank
  int64_t* red_i;  // [kPlaceWaves]
  double* red_d;   // [3 * kPlaceWaves]
};

__host__ __device__ inline size_t align16(size_t v) { return (v + 15) & ~static_cast<size_t>(15); }

// Byte offsets of the LDS carve; the same function sizes the launch.
__host__ __device__ inline size_t place_lds_layout(int S, int E, int G, int chunk, size_t* off) {
  size_t o = 0;
  off[0] = o; o = align16(o + sizeof(int64_t) * E);               // B
  off[1] = o; o = align16(o + sizeof(int64_t) * E);               // V
  off[2] = o; o = align16(o + sizeof(double) * S * G);            // D
  off[3] = o; o = align16(o + sizeof(double2) * chunk * G);       // terms
  off[4] = o; o = align16(o + sizeof(double2) * E);               // won
  off[5] = o; o = align16(o + sizeof(int64_t) * E);               // bo
  off[6] = o; o = align16(o + sizeof(int32_t) * E);               // order
  off[7] = o; o = align16(o + sizeof(int32_t) * E);               // home
  off[8] = o; o = align16(o + sizeof(int32_t) * E);               // xs
  off[9] = o; o = align16(o + sizeof(int32_t) * kPlaceMaxRanks);  // fill
  off[10] = o; o = align16(o + sizeof(int64_t) * kPlaceWaves);    // red_i
  off[11] = o; o = align16(o + sizeof(double) * 3 * kPlaceWaves); // red_d
  return o;
}

__device__ __forceinline__ double mig_cost(const PlaceKernelArgs& a, int l, int e, int g) {
  return a.M ? a.M[(static_cast<size_t>(l) * a.E + e) * a.G + g] : a.m_uniform;
}

// Candidate (score, key) a beats b.  key: bit 31 = rank full, bit 30 = not
// the expert's current rank, bits 6..16 = experts placed, bits 0..5 = rank.
__device__ __forceinline__ bool beats(double as, uint32_t ak, double bs, uint32_t bk) {
  const uint32_t a_full = ak >> 31, b_full = bk >> 31;
  if (a_full != b_full) return a_full < b_full;
  if (as != bs) return as < bs;
  return (ak & 0x7fffffffu) < (bk & 0x7fffffffu);
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

  size_t off[12];
  place_lds_layout(S, E, G, a.chunk, off);
  PlaceLds s;
  s.B = reinterpret_cast<int64_t*>(place_smem + off[0]);
  s.V = reinterpret_cast<int64_t*>(place_smem + off[1]);
  s.D = reinterpret_cast<double*>(place_smem + off[2]);
  s.terms = reinterpret_cast<double2*>(place_smem + off[3]);
  s.won = reinterpret_cast<double2*>(place_smem + off[4]);
  s.bo = reinterpret_cast<int64_t*>(place_smem + off[5]);
  s.order = reinterpret_cast<int32_t*>(place_smem + off[6]);
  s.home = reinterpret_cast<int32_t*>(place_smem + off[7]);
  s.xs = reinterpret_cast<int32_t*>(place_smem + off[8]);
  s.fill = reinterpret_cast<int32_t*>(place_smem + off[9]);
  s.red_i = reinterpret_cast<int64_t*>(place_smem + off[10]);
  s.red_d = reinterpret_cast<double*>(place_smem + off[11]);

  // 1. hotness signals, current ranks, D
  int64_t part = 0;
  for (int e = tid; e < E; e += kPlaceThreads) {
    int64_t v = 0;
    for (int src = 0; src < S; ++src) v += A_l[static_cast<size_t>(src) * E + e];
    const int64_t b = a.B ? a.B[static_cast<size_t>(l) * E + e] : v;
    s.V[e] = v;
    s.B[e] = b;
    s.home[e] = a.x0[static_cast<size_t>(l) * E + e];
    part += b;
  }
  for (int i = tid; i < S * G; i += kPlaceThreads) s.D[i] = a.D[i];
  part = wave_sum_i64(part);
  if (lane == 0) s.red_i[wave] = part;
  __syncthreads();
  int64_t total = 0;
  for (int w = 0; w < kPlaceWaves; ++w) total += s.red_i[w];
  // every expert is placed, so the final average rank load is known up front
  const double mean = static_cast<double>(total) / G;

  // 2. hotness order: position = number of experts that come first
  for (int e = tid; e < E; e += kPlaceThreads) {
    const int64_t be = s.B[e], ve = s.V[e];
    int pos = 0;
    for (int f = 0; f < E; ++f) {
      const int64_t bf = s.B[f], vf = s.V[f];
      pos += (bf > be) || (bf == be && (vf > ve || (vf == ve && f < e)));
    }
    s.order[pos] = e;
    s.bo[pos] = be;
  }
  __syncthreads();

  // 3. greedy, hottest first; wave 0 lane g keeps rank g's state
  int placed = 0;
  int64_t load = 0;
  const int cap_g = lane < G ? a.cap[lane] : 0;
  int span = 1;
  while (span < G) span <<= 1;
  for (int c0 = 0; c0 < E; c0 += a.chunk) {
    const int nc = min(a.chunk, E - c0);
    for (int p = tid; p < nc * G; p += kPlaceThreads) {
      const int i = p / G;
      const int g = p - i * G;
      const int e = s.order[c0 + i];
      double comm = 0.0;
      for (int src = 0; src < S; ++src)
        comm = comm + static_cast<double>(A_l[static_cast<size_t>(src) * E + e]) * s.D[src * G + g];
      const int home = s.home[e];
      const bool home_ok = home >= 0 && home < G;
      double mig = 0.0;
      if (!(home_ok && g == home)) {
        mig = mig_cost(a, l, e, g);
        if (home_ok) mig = mig + mig_cost(a, l, e, home);
      }
      s.terms[p] = make_double2(comm, mig);
    }
    __syncthreads();
    if (wave == 0) {
      for (int i = 0; i < nc; ++i) {
        const int e = s.order[c0 + i];
        const int64_t be = s.bo[c0 + i];
        const int home = s.home[e];
        const bool open = lane < G && placed < cap_g;
        double score = __builtin_inf();
        double2 t = make_double2(0.0, 0.0);
        if (open) {
          t = s.terms[i * G + lane];
          const double u = static_cast<double>(load) - mean;
          const double v = static_cast<double>(load + be) - mean;
          const double c_load = v * v - u * u;
          score = a.alpha * t.x;
          score = score + a.beta * c_load;
          score = score + a.gamma * t.y;
          if (score != score) score = __builtin_inf();
        }
        uint32_t key = (open ? 0u : 0x80000000u) | (lane == home ? 0u : 0x40000000u) |
                       (static_cast<uint32_t>(placed) << 6) | static_cast<uint32_t>(lane);
        for (int o = 1; o < span; o <<= 1) {
          const double os = __shfl_xor(score, o);
          const uint32_t ok = __shfl_xor(key, o);
          if (beats(os, ok, score, key)) {
            score = os;
            key = ok;
          }
        }
        const int w = static_cast<int>(__builtin_amdgcn_readfirstlane(key) & 63u);
        if (lane == w) {
          placed += 1;
          load += be;
          s.xs[e] = w;
          s.won[e] = t;
        }
      }
    }
    __syncthreads();
  }

  // 4. results
  if (wave == 0) {
    if (lane < G) s.fill[lane] = placed;
    if (a.cost) {
      const double d = lane < G ? static_cast<double>(load) - mean : 0.0;
      const double c_load = wave_sum_f64(d * d);
      if (lane == 0) a.cost[static_cast<size_t>(l) * 3 + 1] = c_load;
    }
  }
  __syncthreads();
  double c_comm = 0.0, c_mig = 0.0;
  for (int e = tid; e < E; e += kPlaceThreads) {
    const int g = s.xs[e];
    a.x[static_cast<size_t>(l) * E + e] = g;
    c_comm = c_comm + s.won[e].x;
    c_mig = c_mig + s.won[e].y;
    if (a.rank_experts) {
      int pos = 0;
      for (int f = 0; f < e; ++f) pos += s.xs[f] == g;
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
  if (a.cost) {
    c_comm = wave_sum_f64(c_comm);
    c_mig = wave_sum_f64(c_mig);
    if (lane == 0) {
      s.red_d[wave] = c_comm;
      s.red_d[kPlaceWaves + wave] = c_mig;
    }
    __syncthreads();
    if (tid == 0) {
      double sc = 0.0, sm = 0.0;
      for (int w = 0; w < kPlaceWaves; ++w) {
        sc = sc + s.red_d[w];
        sm = sm + s.red_d[kPlaceWaves + w];
      }
      a.cost[static_cast<size_t>(l) * 3 + 0] = sc;
      a.cost[static_cast<size_t>(l) * 3 + 2] = sm;
    }
  }
}

}  // namespace

int place_chunk(int E, int G) { return min(E, max(1, kChunkTerms / G)); }

size_t place_lds_bytes(int S, int E, int G) {
  size_t off[12];
  return place_lds_layout(S, E, G, place_chunk(E, G), off);
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
  a.chunk = place_chunk(h.E, h.G);
  for (int g = 0; g < h.G; ++g) a.cap[g] = h.cap[g];
  const size_t lds = place_lds_bytes(h.S, h.E, h.G);
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&place_kernel),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, kPlaceMaxLdsBytes);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  hipLaunchKernelGGL(place_kernel, dim3(h.L), dim3(kPlaceThreads), lds, st, a);
  return hipGetLastError();
}

}  // namespace moe
