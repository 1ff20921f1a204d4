// Expert FFN for decode-sized batches: weight streaming.
//
// With at most a few dozen rows per expert the grouped GEMM is bound by
// reading the active experts' weights from HBM exactly once.  The weights take
// the MFMA's 32-row A operand and the tokens its 32-column B operand:
// v_mfma_f32_32x32x16_bf16 computes C[n][t] += W[n][k] X[t][k].
//
// Work split: one workgroup per (expert group, row block).  Its KP waves are
// autonomous: wave p streams K part p of NB weight blocks of 32 rows that
// share the token operand (gate/up: the gate rows and the up rows of the
// same 32 output columns; down: NB consecutive 32-row blocks), in steps of
// KS elements, so every token fragment read from L2 feeds NB MFMAs.  A step
// of a block (32 rows x KS) is loaded by buffer_load_dwordx4 ... lds straight
// into the wave's own ring of two step buffers in LDS; one load instruction
// covers 64/(KS/8) whole rows of KS/8 16-byte pieces, so every request is a
// full run of 128-byte lines.  Piece c of row r lands in slot c ^ (r mod KS/8),
// which spreads the 32 rows of an MFMA fragment read over the banks.  The
// next step's weights stay in flight per wave without holding registers,
// its token fragments in registers.  No workgroup
// barrier is taken inside the K loop; one barrier at the end reduces the K
// parts (fixed order, deterministic) and applies SwiGLU.  Each workgroup
// starts its K walk at a rotated step so that concurrently running
// workgroups, whose rows sit H*2 bytes apart, spread over the HBM channels.
#include "common.h"
#include "ffn_impl.h"

namespace moe {
namespace {

constexpr uint32_t kInvalidOff = 0x80000000u;  // past the descriptor's range: reads zeros, no traffic

// 64 lanes x 16 bytes from rs + off[lane] to lds + 16 * lane.
__device__ __forceinline__ void stream_lds16(__amdgpu_buffer_rsrc_t rs, unsigned char* lds, uint32_t off) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (__attribute__((address_space(3))) void*)lds, 16, off, 0, 0, 0);
}

template <bool GATED, int NB, int KP, int KS, int DEPTH>
__global__ __launch_bounds__(KP* kWave) __attribute__((amdgpu_waves_per_eu(2, 2))) void skinny_kernel(GemmArgs a) {
  constexpr int ROWB = KS * 2;            // bytes of one row segment
  constexpr int PPR = KS / 8;             // 16-byte pieces per row segment
  constexpr int RPI = kWave / PPR;        // rows per load instruction
  constexpr int NLD = 32 / RPI;           // load instructions per block step
  constexpr int KK = KS / 16;             // MFMA k-steps per step
  constexpr int STEPB = 32 * ROWB;        // bytes of one block step
  constexpr int WG_ROWS = GATED ? 32 : 32 * NB;  // output columns of the workgroup
  static_assert(RPI * PPR == kWave && NLD * RPI == 32 && RPI * ROWB == 1024, "step shape");
  // two-step rings: the waits below count the loads of exactly one step ahead
  static_assert(DEPTH == 2 && (!GATED || NB == 2), "ring depth / gated blocks");
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];

  const int g = blockIdx.y;
  int row_base = 0, m = a.static_rows;
  if (a.offsets) {
    row_base = a.offsets[g];
    m = a.offsets[g + 1] - row_base;
  }
  if (m <= 0) return;  // an expert with no rows costs no weight traffic
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave), lane = lane_id();
  // first chunk of this group in the chunk-blocked layouts: the chunks of the
  // groups before it (every wave, lanes over groups)
  int chunk_base = 0;
  if (a.x_blocked || a.out_blocked) {
    for (int g0 = 0; g0 < g; g0 += kWave) {
      const int gg = g0 + lane;
      int c = gg < g ? ceil_div(a.offsets[gg + 1] - a.offsets[gg], kChunkRows) : 0;
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) c += __shfl_xor(c, off);
      chunk_base += c;
    }
  }

  const int part = wave;
  const int n0 = blockIdx.x * WG_ROWS;
  const int nks = ceil_div(a.K, KS);
  const int q0 = part * nks / KP, q1 = (part + 1) * nks / KP;
  const int nq = q1 - q0;
  const int rot = nq > 0 ? static_cast<int>((blockIdx.x * 7u + blockIdx.y * 3u) % nq) : 0;
  unsigned char* wl = smem + wave * (DEPTH * NB * STEPB);  // this wave's ring

  const size_t gofs = static_cast<size_t>(g) * a.group_stride;
  // descriptors of the first (gate, or the only) matrix and the up matrix;
  // plain scalars captured by the load lambda
  const __amdgpu_buffer_rsrc_t rs0 =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(a.w0 + gofs), 0, 0x7fffffff, 0x00020000);
  const __amdgpu_buffer_rsrc_t rs1 =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>((GATED ? a.w1 : a.w0) + gofs), 0, 0x7fffffff, 0x00020000);
  // load i of block b, lane L: row RPI*i + L/PPR of the block, LDS slot L%PPR,
  // global piece slot ^ (row mod PPR)
  uint32_t roff[NB][NLD];
  int piece[NLD];
#pragma unroll
  for (int i = 0; i < NLD; ++i) {
    const int r = RPI * i + lane / PPR;
    piece[i] = (lane % PPR) ^ (r & (PPR - 1));
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const int n = n0 + (GATED ? 0 : 32 * b) + r;
      roff[b][i] = n < a.N ? static_cast<uint32_t>(n * a.ldw * 2) : kInvalidOff;
    }
  }
  const bool segmented = a.kseg < a.K;

  auto kstep = [&](int j) {
    int s = rot + j;
    if (s >= nq) s -= nq;
    return q0 + s;
  };
  // the weights of step j into ring slot j % DEPTH
  auto issue = [&](int j) {
    const int kk0 = kstep(j) * KS;
    unsigned char* dst = wl + (j % DEPTH) * (NB * STEPB);
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      // every load is issued (the wait counts rely on it): a piece past K
      // gets an offset past the descriptor's range
      const int kk = kk0 + piece[i] * 8;
      const bool kok = kk < a.K;
      const int kc = kok ? kk : kk0;
      const uint32_t col = static_cast<uint32_t>((segmented ? weight_col_offset(a, kc) : static_cast<size_t>(kc)) * 2);
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const uint32_t off = (roff[b][i] + col) | (kok ? 0u : kInvalidOff);
        if (GATED && b == 1)
          stream_lds16(rs1, dst + b * STEPB + i * 1024, off);
        else
          stream_lds16(rs0, dst + b * STEPB + i * 1024, off);
      }
    }
  };

  for (int tok0 = 0; tok0 < m; tok0 += 64) {
    const int mc = min(64, m - tok0);
    const int nch = mc > 32 ? 2 : 1;
    // per chunk: the lane's 16 bytes of the step's first MFMA B operand; the
    // following K-steps sit kstride elements further
    const uint16_t* xrow[2];
    bool tok_ok[2];
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int tok = tok0 + c * 32 + (lane & 31);
      if (a.x_blocked) {  // chunk rows past m are zeros
        tok_ok[c] = c < nch;
        xrow[c] = a.x + static_cast<size_t>(chunk_base + tok0 / kChunkRows + c) * (a.K / 16) * kBlockElems + lane * 8;
      } else {
        tok_ok[c] = c < nch && tok < m;
        const int r = row_base + (tok_ok[c] ? tok : 0);
        xrow[c] = a.x + static_cast<size_t>(a.x_rows ? a.x_rows[r] : r) * a.K + 8 * (lane >> 5);
      }
    }
    const int kstride = a.x_blocked ? kBlockElems : 16;  // elements between consecutive 16-wide K-steps

    f32x16 acc[NB][2];
#pragma unroll
    for (int b = 0; b < NB; ++b) acc[b][0] = acc[b][1] = f32x16{};
    if constexpr (GATED) {
      // The token fragments of step j + 1 (2 KK loads into the other of two
      // register sets; always issued, a lane out of range reading its row's
      // first piece) go out before the weights of step j + 1, so that both are
      // in flight while step j computes.  Pieces out of range are zeroed after
      // the wait.
      u32x4 xs[2][2][KK];
      auto x_ok = [&](int kb, int c, int kk) {
        return tok_ok[c] && kb * KS + 16 * kk + 8 * (lane >> 5) < a.K;
      };
      // chunk 1 only when the row block has a second chunk (uniform)
      auto load_x = [&](int j, u32x4 (&dst)[2][KK]) {
        const int kb = kstep(j);
#pragma unroll
        for (int c = 0; c < 2; ++c) {
          if (c == 1 && nch < 2) break;
#pragma unroll
          for (int kk = 0; kk < KK; ++kk)
            dst[c][kk] = load16(xrow[c] + (x_ok(kb, c, kk) ? (kb * (KS / 16) + kk) * kstride : 0));
        }
      };
      auto step = [&](int j, u32x4 (&cur)[2][KK], u32x4 (&nxt)[2][KK]) {
        // the slot refilled is the one step j-1 read, whose fragments are in
        // registers by now
        if (j + 1 < nq) {
          load_x(j + 1, nxt);
          issue(j + 1);
          // step j + 1's loads may stay in flight
          constexpr int kYounger2 = 2 * KK + NB * NLD, kYounger1 = KK + NB * NLD;
          if (nch > 1)
            __builtin_amdgcn_s_waitcnt((kYounger2 & 15) | ((kYounger2 >> 4) << 14) | (7 << 4) | (15 << 8));
          else
            __builtin_amdgcn_s_waitcnt((kYounger1 & 15) | ((kYounger1 >> 4) << 14) | (7 << 4) | (15 << 8));
        } else {
          __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));  // vmcnt(0)
        }
        const int kb = kstep(j);
#pragma unroll
        for (int c = 0; c < 2; ++c)
#pragma unroll
          for (int kk = 0; kk < KK; ++kk) {
            const u32x4 zero = {0u, 0u, 0u, 0u};
            if (!x_ok(kb, c, kk)) cur[c][kk] = zero;
          }
        const unsigned char* bsl = wl + (j % DEPTH) * (NB * STEPB);
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
          const int p = 2 * kk + (lane >> 5);
          const int row = lane & 31;
          const int slot = row * ROWB + ((p ^ (row & (PPR - 1))) << 4);
#pragma unroll
          for (int b = 0; b < NB; ++b) {
            const u32x4 wv = *reinterpret_cast<const u32x4*>(bsl + b * STEPB + slot);
            acc[b][0] = mfma32x32x16(as_bf16x8(wv), as_bf16x8(cur[0][kk]), acc[b][0]);
            if (nch > 1) acc[b][1] = mfma32x32x16(as_bf16x8(wv), as_bf16x8(cur[1][kk]), acc[b][1]);
          }
        }
      };
      if (nq > 0) {
        load_x(0, xs[0]);
        issue(0);
      }
      for (int j = 0; j < nq; j += 2) {
        step(j, xs[0], xs[1]);
        if (j + 1 < nq) step(j + 1, xs[1], xs[0]);
      }
    } else {
      // down: step j's token fragments just before the weights of step j + 1
      // (measured faster here than one step ahead)
      for (int s = 0; s < DEPTH - 1; ++s)
        if (s < nq) issue(s);
      for (int j = 0; j < nq; ++j) {
        const int kb = kstep(j);
        u32x4 xt[2][KK];
#pragma unroll
        for (int c = 0; c < 2; ++c)
#pragma unroll
          for (int kk = 0; kk < KK; ++kk) {
            const int k = kb * KS + 16 * kk + 8 * (lane >> 5);
            const u32x4 zero = {0u, 0u, 0u, 0u};
            xt[c][kk] = (tok_ok[c] && k < a.K) ? load16(xrow[c] + (kb * (KS / 16) + kk) * kstride) : zero;
          }
        // keep DEPTH-1 steps in flight; the slot refilled is the one step j-1
        // read, whose fragments are in registers by now
        if (j + DEPTH - 1 < nq) {
          issue(j + DEPTH - 1);
          constexpr int kYounger = NB * NLD;  // the loads just issued may stay in flight
          __builtin_amdgcn_s_waitcnt((kYounger & 15) | ((kYounger >> 4) << 14) | (7 << 4) | (15 << 8));
        } else {
          __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));  // vmcnt(0)
        }
        const unsigned char* bsl = wl + (j % DEPTH) * (NB * STEPB);
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
          const int p = 2 * kk + (lane >> 5);
          const int row = lane & 31;
          const int slot = row * ROWB + ((p ^ (row & (PPR - 1))) << 4);
#pragma unroll
          for (int b = 0; b < NB; ++b) {
            const u32x4 wv = *reinterpret_cast<const u32x4*>(bsl + b * STEPB + slot);
            acc[b][0] = mfma32x32x16(as_bf16x8(wv), as_bf16x8(xt[0][kk]), acc[b][0]);
            if (nch > 1) acc[b][1] = mfma32x32x16(as_bf16x8(wv), as_bf16x8(xt[1][kk]), acc[b][1]);
          }
        }
      }
    }

    // reduce the K parts in a fixed order; wave 0 applies the epilogue
    __syncthreads();
    float* red = reinterpret_cast<float*>(smem);
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int c = 0; c < 2; ++c)
        if (c < nch)
#pragma unroll
          for (int v = 0; v < 16; ++v) red[(((wave * NB + b) * 2 + c) * 16 + v) * kWave + lane] = acc[b][c][v];
    __syncthreads();
    if (wave == 0) {
      // lane holds C[n = 8*(v/4) + 4*(lane/32) + v%4][t = lane%32] of each chunk
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const int tok = tok0 + c * 32 + (lane & 31);
        if (c >= nch || (!a.out_blocked && tok >= m)) continue;
        uint16_t* orow = a.out + static_cast<size_t>(row_base + tok) * a.N;
        uint16_t* oblk = a.out + static_cast<size_t>(chunk_base + tok0 / kChunkRows + c) * (a.N / 16) * kBlockElems +
                         8 * (lane & 31);
        constexpr int NOUT = GATED ? 1 : NB;  // 32-column output blocks
#pragma unroll
        for (int ob = 0; ob < NOUT; ++ob)
#pragma unroll
          for (int v4 = 0; v4 < 4; ++v4) {
            const int n = n0 + 32 * ob + 8 * v4 + 4 * (lane >> 5);
            if (n >= a.N) continue;
            float o[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int v = 4 * v4 + i;
              float s0 = 0.f, s1 = 0.f;
              for (int p = 0; p < KP; ++p) s0 += red[(((p * NB + (GATED ? 0 : ob)) * 2 + c) * 16 + v) * kWave + lane];
              if (GATED)
                for (int p = 0; p < KP; ++p) s1 += red[(((p * NB + 1) * 2 + c) * 16 + v) * kWave + lane];
              o[i] = GATED ? silu(s0) * s1 : s0;
            }
            uint2 pk;
            pk.x = pack_bf16x2(o[0], o[1]);
            pk.y = pack_bf16x2(o[2], o[3]);
            // blocked: columns n..n+3 of row t go to block n/16, lane 32*((n/8)&1) + t, values n%8..
            uint16_t* dst = a.out_blocked ? oblk + (n >> 4) * kBlockElems + 256 * ((n >> 3) & 1) + (n & 7) : orow + n;
            *reinterpret_cast<uint2*>(dst) = pk;
          }
      }
    }
    __syncthreads();
  }
}

template <bool GATED, int NB, int KP, int KS, int DEPTH>
hipError_t launch_skinny_t(const Segments& seg, const GemmArgs& a, hipStream_t st) {
  constexpr size_t kRing = static_cast<size_t>(KP) * DEPTH * NB * 32 * KS * 2;
  constexpr size_t kRed = static_cast<size_t>(KP) * NB * 2 * 16 * kWave * 4;
  constexpr size_t kLds = kRing > kRed ? kRing : kRed;
  static_assert(kLds <= 160 * 1024, "LDS");
  constexpr int WG_ROWS = GATED ? 32 : 32 * NB;
  static unsigned long long lds_set = 0;  // devices with the LDS limit raised
  const hipError_t e_lds =
      set_max_dynamic_lds(reinterpret_cast<const void*>(&skinny_kernel<GATED, NB, KP, KS, DEPTH>),
                          static_cast<int>(kLds), &lds_set);
  if (e_lds != hipSuccess) return e_lds;
  dim3 grid(ceil_div(a.N, WG_ROWS), seg.groups);
  hipLaunchKernelGGL((skinny_kernel<GATED, NB, KP, KS, DEPTH>), grid, dim3(KP * kWave), kLds, st, a);
  return hipGetLastError();
}

}  // namespace

size_t chunk_capacity(int groups, int total_rows) {
  return static_cast<size_t>(total_rows / kChunkRows) + static_cast<size_t>(std::min(groups, total_rows));
}

bool skinny_ok(const GemmArgs& a) {
  if ((a.x_blocked || a.out_blocked) && (a.K % 16 != 0 || (a.out_blocked && a.N % 16 != 0))) return false;
  // weight byte offsets within a group are 32-bit
  const size_t w_span = (static_cast<size_t>(a.N) * a.ldw +
                         (a.kseg < a.K ? static_cast<size_t>((a.K - 1) / a.kseg) * a.seg_stride : 0) + a.K) * 2;
  return w_span < kInvalidOff;
}

hipError_t launch_skinny(const Segments& seg, const GemmArgs& a, bool gated, hipStream_t st) {
  // the blocked layouts are defined by the device-side offsets
  if ((a.x_blocked || a.out_blocked) && a.offsets == nullptr) return hipErrorInvalidValue;
  // the gate/up kernel's out-of-range token lanes read their row's first
  // piece, which exists only in the row layout
  if (gated && a.x_blocked) return hipErrorInvalidValue;
  if (!skinny_ok(a)) return hipErrorInvalidValue;
  // gate/up: the gate and up blocks of 32 rows per wave; down: two 32-row
  // blocks per wave; 4 K parts, 64-wide steps, two-step rings (64 KB of LDS,
  // two workgroups per CU): the measured best shapes for the decode workload
  return gated ? launch_skinny_t<true, 2, 4, 64, 2>(seg, a, st) : launch_skinny_t<false, 2, 4, 64, 2>(seg, a, st);
}

}  // namespace moe
