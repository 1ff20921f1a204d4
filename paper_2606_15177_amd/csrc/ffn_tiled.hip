// Expert FFN for prefill-sized batches: a persistent, LDS-tiled bf16 MFMA
// grouped GEMM.
//
// Output tiles are BM token rows x BN weight rows of one group (expert).  The
// tile list is implied by the device-side offsets: every workgroup computes
// the per-group prefix of ceil(rows/BM) once, then walks tile ids
// blockIdx', blockIdx'+gridDim, ... where blockIdx' renumbers workgroups so
// that each XCD (workgroups are dealt round-robin to the 8 XCDs) owns a
// contiguous run of tiles: consecutive tiles share the token rows and, within
// one expert, the weights, which keeps them in that XCD's L2.  Group sizes
// never leave the device.
//
// K loop: BK = 64.  Each K-block of X (BM x 64) and W (BN x 64) is loaded
// with 16-byte vectors into registers, then stored to one of two LDS buffers
// (row = 128 bytes, 16-byte chunk c of row r stored at slot c ^ (r & 7), so
// the MFMA fragment reads of 8 consecutive rows hit distinct banks).  The
// load of block kb+1 is in flight while block kb feeds the MFMAs.
//
// MFMA v_mfma_f32_32x32x16_bf16 with the weights as the A operand and tokens
// as B: C[n][t]; lane l then holds 4 consecutive output columns of token
// l % 32 in each group of 4 accumulators, written as one 8-byte store.  For
// the gate/up GEMM the BN weight rows of a wave are its WTN/2 gate rows
// followed by the WTN/2 up rows of the same columns, so each lane holds
// gate and up for the same (token, column) and applies SwiGLU in registers.
#include "ffn_impl.h"

namespace moe {
namespace {

constexpr int kBK = 64;
constexpr int kMaxGroups = 1024;

template <int BM, int BN, int WM, int WN, bool GATED>
__global__ __launch_bounds__(WM* WN* kWave) void tiled_kernel(GemmArgs a) {
  constexpr int kThreads = WM * WN * kWave;
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  constexpr int X_CH = BM * 8 / kThreads;
  constexpr int W_CH = BN * 8 / kThreads;
  constexpr int kXBytes = BM * 128;
  constexpr int kBufBytes = (BM + BN) * 128;
  constexpr int OUT_COLS = GATED ? BN / 2 : BN;
  static_assert(TM >= 1 && TN >= 1 && (!GATED || TN % 2 == 0), "tile shape");
  static_assert(X_CH * kThreads == BM * 8 && W_CH * kThreads == BN * 8, "chunking");

  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  __shared__ int mt_prefix[kMaxGroups + 1];

  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wave = tid / kWave;
  const int wm = wave % WM, wn = wave / WM;
  const int lrow = lane & 31, lhalf = lane >> 5;
  const int n_tiles_n = ceil_div(a.N, OUT_COLS);

  int total_mt;
  if (a.offsets == nullptr) {
    total_mt = ceil_div(a.static_rows, BM);
  } else {
    if (wave == 0) {
      int carry = 0;
      for (int g0 = 0; g0 < a.groups; g0 += kWave) {
        const int g = g0 + lane;
        const int cnt = g < a.groups ? ceil_div(a.offsets[g + 1] - a.offsets[g], BM) : 0;
        int inc = cnt;
#pragma unroll
        for (int off = 1; off < kWave; off <<= 1) {
          const int o = __shfl_up(inc, off);
          if (lane >= off) inc += o;
        }
        if (g < a.groups) mt_prefix[g] = carry + inc - cnt;
        carry += __shfl(inc, kWave - 1);
      }
      if (lane == 0) mt_prefix[a.groups] = carry;
    }
    __syncthreads();
    total_mt = mt_prefix[a.groups];
  }
  const int total_tiles = total_mt * n_tiles_n;

  // XCD-aware renumbering (gridDim.x is a multiple of 8)
  const int per_xcd = gridDim.x / 8;
  const int vblock = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;

  // fixed per-thread chunk coordinates
  const int cc = tid & 7;  // 16-byte chunk within a 128-byte row (same for all i)
  int x_lds[X_CH], w_lds[W_CH];
#pragma unroll
  for (int i = 0; i < X_CH; ++i) {
    const int r = (tid >> 3) + i * (kThreads / 8);
    x_lds[i] = r * 128 + ((cc ^ (r & 7)) << 4);
  }
#pragma unroll
  for (int i = 0; i < W_CH; ++i) {
    const int n = (tid >> 3) + i * (kThreads / 8);
    w_lds[i] = kXBytes + n * 128 + ((cc ^ (n & 7)) << 4);
  }
  const int nkb = ceil_div(a.K, kBK);

  for (int tile = vblock; tile < total_tiles; tile += gridDim.x) {
    const int mt = tile / n_tiles_n;
    const int nt = tile - mt * n_tiles_n;
    int g = 0, row_base = 0, m = a.static_rows, m0 = mt * BM;
    if (a.offsets != nullptr) {
      int lo = 0, hi = a.groups - 1;
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (mt_prefix[mid] <= mt) lo = mid; else hi = mid - 1;
      }
      g = lo;
      row_base = a.offsets[g];
      m = a.offsets[g + 1] - row_base;
      m0 = (mt - mt_prefix[g]) * BM;
    }

    const uint16_t* xsrc[X_CH];
    bool xok[X_CH];
#pragma unroll
    for (int i = 0; i < X_CH; ++i) {
      const int r = m0 + (tid >> 3) + i * (kThreads / 8);
      xok[i] = r < m;
      xsrc[i] = a.x + static_cast<size_t>(row_base + (xok[i] ? r : 0)) * a.K + cc * 8;
    }
    const uint16_t* wsrc[W_CH];
    bool wok[W_CH];
#pragma unroll
    for (int i = 0; i < W_CH; ++i) {
      const int n = (tid >> 3) + i * (kThreads / 8);
      int col;
      const uint16_t* base;
      if constexpr (GATED) {
        const int wn_ = n / WTN, within = n % WTN;
        col = nt * OUT_COLS + wn_ * (WTN / 2) + within % (WTN / 2);
        base = (within >= WTN / 2) ? a.w1 : a.w0;
      } else {
        col = nt * BN + n;
        base = a.w0;
      }
      wok[i] = col < a.N;
      wsrc[i] = base + static_cast<size_t>(g) * a.group_stride +
                static_cast<size_t>(wok[i] ? col : 0) * a.ldw;
    }

    u32x4 rx[X_CH], rw[W_CH];
    auto load_block = [&](int kb) {
      const int kk = kb * kBK + cc * 8;
      const bool kok = kk < a.K;
      const size_t wc = kok ? weight_col_offset(a, kk) : 0;
      const u32x4 zero = {0u, 0u, 0u, 0u};
#pragma unroll
      for (int i = 0; i < X_CH; ++i) rx[i] = (kok && xok[i]) ? load16(xsrc[i] + kb * kBK) : zero;
#pragma unroll
      for (int i = 0; i < W_CH; ++i) rw[i] = (kok && wok[i]) ? load16(wsrc[i] + wc) : zero;
    };
    auto store_block = [&](int buf) {
      unsigned char* b = smem + buf * kBufBytes;
#pragma unroll
      for (int i = 0; i < X_CH; ++i) *reinterpret_cast<u32x4*>(b + x_lds[i]) = rx[i];
#pragma unroll
      for (int i = 0; i < W_CH; ++i) *reinterpret_cast<u32x4*>(b + w_lds[i]) = rw[i];
    };

    f32x16 acc[TN][TM];
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
#pragma unroll
      for (int tm = 0; tm < TM; ++tm) acc[tn][tm] = f32x16{};

    load_block(0);
    store_block(0);
    __syncthreads();
    for (int kb = 0; kb < nkb; ++kb) {
      const int buf = kb & 1;
      if (kb + 1 < nkb) load_block(kb + 1);
      const unsigned char* b = smem + buf * kBufBytes;
#pragma unroll
      for (int ks = 0; ks < kBK / 16; ++ks) {
        const int ch = 2 * ks + lhalf;
        bf16x8 wf[TN], xf[TM];
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) {
          const int n = wn * WTN + tn * 32 + lrow;
          wf[tn] = as_bf16x8(*reinterpret_cast<const u32x4*>(b + kXBytes + n * 128 + ((ch ^ (n & 7)) << 4)));
        }
#pragma unroll
        for (int tm = 0; tm < TM; ++tm) {
          const int r = wm * WTM + tm * 32 + lrow;
          xf[tm] = as_bf16x8(*reinterpret_cast<const u32x4*>(b + r * 128 + ((ch ^ (r & 7)) << 4)));
        }
#pragma unroll
        for (int tn = 0; tn < TN; ++tn)
#pragma unroll
          for (int tm = 0; tm < TM; ++tm) acc[tn][tm] = mfma32x32x16(wf[tn], xf[tm], acc[tn][tm]);
      }
      if (kb + 1 < nkb) store_block(buf ^ 1);
      __syncthreads();
    }

    // epilogue: lane holds C[n = 8*(v/4) + 4*lhalf + v%4][t = lrow] per 32x32 tile
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) {
      const int row = m0 + wm * WTM + tm * 32 + lrow;
      if (row >= m) continue;
      uint16_t* orow = a.out + static_cast<size_t>(row_base + row) * a.N;
      constexpr int TOUT = GATED ? TN / 2 : TN;
#pragma unroll
      for (int tn = 0; tn < TOUT; ++tn) {
#pragma unroll
        for (int v4 = 0; v4 < 4; ++v4) {
          const int col = GATED ? nt * OUT_COLS + wn * (WTN / 2) + tn * 32 + 8 * v4 + 4 * lhalf
                                : nt * BN + wn * WTN + tn * 32 + 8 * v4 + 4 * lhalf;
          if (col >= a.N) continue;
          float o[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float c0 = acc[tn][tm][4 * v4 + i];
            if constexpr (GATED)
              o[i] = silu(c0) * acc[tn + TN / 2][tm][4 * v4 + i];
            else
              o[i] = c0;
          }
          uint2 pk;
          pk.x = pack_bf16x2(o[0], o[1]);
          pk.y = pack_bf16x2(o[2], o[3]);
          *reinterpret_cast<uint2*>(orow + col) = pk;
        }
      }
    }
  }
}

int device_cu_count() {
  static int cus = 0;
  if (cus == 0) {
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && n > 0)
      cus = n;
    else
      cus = 256;
  }
  return cus;
}

template <int BM, int BN, int WM, int WN, bool GATED>
hipError_t launch_tiled_t(const Segments& seg, const GemmArgs& a, hipStream_t st) {
  constexpr int kThreads = WM * WN * kWave;
  constexpr int OUT_COLS = GATED ? BN / 2 : BN;
  constexpr size_t kLds = 2 * (BM + BN) * 128;
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&tiled_kernel<BM, BN, WM, WN, GATED>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(kLds));
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  const long long m_tiles = (a.offsets ? static_cast<long long>(ceil_div(seg.total_rows, BM)) + seg.groups
                                       : ceil_div(seg.static_rows, BM));
  const long long tiles = m_tiles * ceil_div(a.N, OUT_COLS);
  if (tiles == 0) return hipSuccess;
  const int wgs_per_cu = 2;
  long long grid = std::min<long long>(tiles, static_cast<long long>(device_cu_count()) * wgs_per_cu);
  grid = ((grid + 7) / 8) * 8;
  hipLaunchKernelGGL((tiled_kernel<BM, BN, WM, WN, GATED>), dim3(static_cast<unsigned>(grid)),
                     dim3(kThreads), kLds, st, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_tiled(const Segments& seg, const GemmArgs& a, bool gated, hipStream_t st) {
  if (seg.groups > kMaxGroups) return hipErrorInvalidValue;
  return gated ? launch_tiled_t<128, 128, 2, 2, true>(seg, a, st)
               : launch_tiled_t<128, 128, 2, 2, false>(seg, a, st);
}

hipError_t launch_ffn_up(const Segments& seg, const UpArgs& u, hipStream_t st) {
  GemmArgs a{};
  a.x = u.x;
  a.offsets = seg.offsets;
  a.static_rows = seg.static_rows;
  a.groups = seg.groups;
  a.w0 = u.w_gate;
  a.w1 = u.w_up;
  a.out = u.h;
  a.K = u.K;
  a.N = u.N;
  a.kseg = u.K;
  a.ldw = u.K;
  a.seg_stride = 0;
  a.group_stride = static_cast<size_t>(u.N) * u.K;
  if (seg.max_rows <= kSkinnyMaxRows) return launch_skinny(seg, a, true, st);
  return launch_tiled(seg, a, true, st);
}

hipError_t launch_ffn_down(const Segments& seg, const DownArgs& d, hipStream_t st) {
  GemmArgs a{};
  a.x = d.h;
  a.offsets = seg.offsets;
  a.static_rows = seg.static_rows;
  a.groups = seg.groups;
  a.w0 = d.w;
  a.w1 = nullptr;
  a.out = d.y;
  a.K = d.K;
  a.N = d.N;
  a.kseg = d.kseg;
  a.ldw = d.ldw;
  a.seg_stride = d.seg_stride;
  a.group_stride = d.group_stride;
  if (seg.max_rows <= kSkinnyMaxRows) return launch_skinny(seg, a, false, st);
  return launch_tiled(seg, a, false, st);
}

}  // namespace moe
