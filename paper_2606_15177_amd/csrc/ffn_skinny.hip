// Expert FFN for decode-sized batches: weight streaming.
//
// With at most a few dozen rows per expert the grouped GEMM is bound by
// reading the active experts' weights from HBM exactly once.  The weights take
// the MFMA's 32-row A operand and the tokens its 32-column B operand:
// v_mfma_f32_32x32x16_bf16 computes C[n][t] += W[n][k] X[t][k].
//
// Work split: one workgroup per (expert group, 32 weight rows).  Its
// NMAT*KP waves are autonomous: wave w streams matrix w / KP (gate or up, or
// the single down matrix) over K part w % KP, in steps of KS elements.  Each
// step is loaded with row-contiguous 16-byte vectors (KS/8 lanes cover one
// row's segment, so every request is a full run of 128-byte lines) into a
// register ring DEPTH steps deep, then transposed through the wave's own LDS
// region into the MFMA operand layout (16-byte slot c of row r stored at
// c ^ (r mod KS/8), so the 32 rows read by one fragment spread over the
// banks).  No workgroup barrier is taken inside the K loop; one barrier at the
// end reduces the K parts (fixed order, deterministic) and applies SwiGLU.
// Each workgroup starts its K walk at a rotated step so that concurrently
// running workgroups, whose rows sit H*2 bytes apart, spread over the HBM
// channels instead of queueing on the same ones.
#include "common.h"
#include "ffn_impl.h"

namespace moe {
namespace {

template <int NMAT, int KP, int KS, int DEPTH>
__global__ __launch_bounds__(NMAT* KP* kWave) void skinny_kernel(GemmArgs a) {
  constexpr int W = NMAT * KP;
  constexpr int ROWB = KS * 2;          // bytes of one row segment
  constexpr int PPR = KS / 8;           // 16-byte pieces per row segment
  constexpr int CPL = 32 * PPR / kWave; // pieces per lane per step
  constexpr int KK = KS / 16;           // MFMA k-steps per step
  static_assert(CPL >= 1 && (kWave % PPR) == 0, "step shape");
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];

  const int g = blockIdx.y;
  int row_base = 0, m = a.static_rows;
  if (a.offsets) {
    row_base = a.offsets[g];
    m = a.offsets[g + 1] - row_base;
  }
  if (m <= 0) return;  // an expert with no rows costs no weight traffic

  const int tid = threadIdx.x, wave = tid / kWave, lane = lane_id();
  const int mat = wave / KP, part = wave % KP;
  const int n0 = blockIdx.x * 32;
  const int nks = ceil_div(a.K, KS);
  const int q0 = part * nks / KP, q1 = (part + 1) * nks / KP;
  const int nq = q1 - q0;
  const int rot = nq > 0 ? static_cast<int>((blockIdx.x * 7u + blockIdx.y * 3u) % nq) : 0;
  unsigned char* wl = smem + wave * (32 * ROWB);

  const uint16_t* wbase = (mat == 0 ? a.w0 : a.w1) + static_cast<size_t>(g) * a.group_stride;
  const int p_l = lane % PPR;
  size_t roff[CPL];
  int dst[CPL];
  bool rok[CPL];
#pragma unroll
  for (int i = 0; i < CPL; ++i) {
    const int r = lane / PPR + (kWave / PPR) * i;
    rok[i] = n0 + r < a.N;
    roff[i] = static_cast<size_t>(rok[i] ? n0 + r : 0) * a.ldw;
    dst[i] = r * ROWB + ((p_l ^ (r & (PPR - 1))) << 4);
  }

  auto kstep = [&](int j) {
    int s = rot + j;
    if (s >= nq) s -= nq;
    return q0 + s;
  };

  for (int tok0 = 0; tok0 < m; tok0 += 64) {
    const int mc = min(64, m - tok0);
    const int nch = mc > 32 ? 2 : 1;
    const uint16_t* xrow[2];
    bool tok_ok[2];
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int tok = tok0 + c * 32 + (lane & 31);
      tok_ok[c] = c < nch && tok < m;
      const int r = row_base + (tok_ok[c] ? tok : 0);
      xrow[c] = a.x + static_cast<size_t>(a.x_rows ? a.x_rows[r] : r) * a.K + 8 * (lane >> 5);
    }

    u32x4 st[DEPTH][CPL];
    f32x16 acc[2] = {f32x16{}, f32x16{}};
    auto gload = [&](u32x4 (&s)[CPL], int kb) {
      const int kk = kb * KS + p_l * 8;
      const bool kok = kk < a.K;
      const size_t col = kok ? weight_col_offset(a, kk) : 0;
      const u32x4 zero = {0u, 0u, 0u, 0u};
#pragma unroll
      for (int i = 0; i < CPL; ++i) s[i] = (rok[i] && kok) ? load16(wbase + roff[i] + col) : zero;
    };

#pragma unroll
    for (int s = 0; s < DEPTH; ++s)
      if (s < nq) gload(st[s], kstep(s));
    for (int j0 = 0; j0 < nq; j0 += DEPTH) {
#pragma unroll
      for (int u = 0; u < DEPTH; ++u) {
        const int j = j0 + u;
        if (j < nq) {
          const int kb = kstep(j);
          u32x4 xt[2][KK];
#pragma unroll
          for (int c = 0; c < 2; ++c)
#pragma unroll
            for (int kk = 0; kk < KK; ++kk) {
              const int k = kb * KS + 16 * kk + 8 * (lane >> 5);
              const u32x4 zero = {0u, 0u, 0u, 0u};
              xt[c][kk] = (tok_ok[c] && k < a.K) ? load16(xrow[c] + kb * KS + 16 * kk) : zero;
            }
#pragma unroll
          for (int i = 0; i < CPL; ++i) *reinterpret_cast<u32x4*>(wl + dst[i]) = st[u][i];
          if (j + DEPTH < nq) gload(st[u], kstep(j + DEPTH));
#pragma unroll
          for (int kk = 0; kk < KK; ++kk) {
            const int p = 2 * kk + (lane >> 5);
            const int row = lane & 31;
            const u32x4 wv =
                *reinterpret_cast<const u32x4*>(wl + row * ROWB + ((p ^ (row & (PPR - 1))) << 4));
            acc[0] = mfma32x32x16(as_bf16x8(wv), as_bf16x8(xt[0][kk]), acc[0]);
            if (nch > 1) acc[1] = mfma32x32x16(as_bf16x8(wv), as_bf16x8(xt[1][kk]), acc[1]);
          }
        }
      }
    }

    // reduce the K parts in a fixed order; wave 0 applies the epilogue
    __syncthreads();
    float* red = reinterpret_cast<float*>(smem);
#pragma unroll
    for (int c = 0; c < 2; ++c)
      if (c < nch)
#pragma unroll
        for (int v = 0; v < 16; ++v) red[((wave * 2 + c) * 16 + v) * kWave + lane] = acc[c][v];
    __syncthreads();
    if (wave == 0) {
      // lane holds C[n = 8*(v/4) + 4*(lane/32) + v%4][t = lane%32] of each chunk
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const int tok = tok0 + c * 32 + (lane & 31);
        if (c >= nch || tok >= m) continue;
        uint16_t* orow = a.out + static_cast<size_t>(row_base + tok) * a.N;
#pragma unroll
        for (int v4 = 0; v4 < 4; ++v4) {
          const int n = n0 + 8 * v4 + 4 * (lane >> 5);
          if (n >= a.N) continue;
          float o[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int v = 4 * v4 + i;
            float s0 = 0.f, s1 = 0.f;
            for (int p = 0; p < KP; ++p) s0 += red[((p * 2 + c) * 16 + v) * kWave + lane];
            if (NMAT == 2)
              for (int p = 0; p < KP; ++p) s1 += red[(((KP + p) * 2 + c) * 16 + v) * kWave + lane];
            o[i] = NMAT == 2 ? silu(s0) * s1 : s0;
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

template <int NMAT, int KP, int KS, int DEPTH>
hipError_t launch_skinny_t(const Segments& seg, const GemmArgs& a, hipStream_t st) {
  constexpr int W = NMAT * KP;
  constexpr size_t kLds = (32 * KS * 2 > 2 * 16 * kWave * 4) ? W * 32 * KS * 2 : W * 2 * 16 * kWave * 4;
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&skinny_kernel<NMAT, KP, KS, DEPTH>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(kLds));
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  dim3 grid(ceil_div(a.N, 32), seg.groups);
  hipLaunchKernelGGL((skinny_kernel<NMAT, KP, KS, DEPTH>), grid, dim3(W * kWave), kLds, st, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_skinny(const Segments& seg, const GemmArgs& a, bool gated, hipStream_t st) {
  // gate/up: 2 matrices x 4 K parts, 64-wide steps; down: 8 K parts, 128-wide
  // steps (the measured best shapes for the decode workload)
  return gated ? launch_skinny_t<2, 4, 64, 2>(seg, a, st) : launch_skinny_t<1, 8, 128, 2>(seg, a, st);
}

}  // namespace moe
