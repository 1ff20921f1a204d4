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
// (row = 128 bytes, 16-byte chunk c of row r stored at slot c ^ swz(r), so
// the MFMA fragment reads spread over all banks).  The
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

// LDS slot key of a 128-byte row: chunk c of row r is stored in slot
// c ^ swz(r).  Among any 16 consecutive rows, each run of 8 and each set of 8
// same-parity rows gets 8 distinct keys, so the 16-byte fragment reads of an
// MFMA operand are bank-conflict free whether the LDS serves 8 or 16 lanes of
// 16 bytes per cycle.  The key depends on r mod 16 only, so writers (which
// know a row modulo their staging stride) and readers (modulo 32) agree.
__device__ __forceinline__ int swz(int r) { return (r & 7) ^ ((r >> 3) & 1); }

// Issue order of one K-block, as scheduling-group constraints on MFMA index
// m = 0..S*P-1 (S steps of P MFMAs, F fragment reads per step): after each
// MFMA, the next step's fragment reads spread evenly over the step; the L
// global loads of the next K-block spread over the first half of the MFMAs
// and its Wn LDS stores over the second half.  The matrix cores are fed
// continuously instead of idling through a load/store burst each block.
template <int m, int S, int P, int F, int L, int Wn>
__device__ __forceinline__ void sched_mfma_seq() {
  if constexpr (m < S * P) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
    constexpr int step = m / P, j = m % P;
    if constexpr (step + 1 < S) {
      constexpr int r0 = F * j / P, r1 = F * (j + 1) / P;
      if constexpr (r1 > r0) __builtin_amdgcn_sched_group_barrier(0x100, r1 - r0, 0);  // LDS reads
    }
    constexpr int H = S * P / 2;
    if constexpr (m < H) {
      constexpr int a = L * m / H, b = L * (m + 1) / H;
      if constexpr (b > a) __builtin_amdgcn_sched_group_barrier(0x020, b - a, 0);  // global loads
    } else {
      constexpr int a = Wn * (m - H) / H, b = Wn * (m - H + 1) / H;
      if constexpr (b > a) __builtin_amdgcn_sched_group_barrier(0x200, b - a, 0);  // LDS stores
    }
    sched_mfma_seq<m + 1, S, P, F, L, Wn>();
  }
}
template <int S, int P, int F, int L, int Wn>
__device__ __forceinline__ void sched_kblock() {
  __builtin_amdgcn_sched_group_barrier(0x100, F, 0);  // step 0's fragment reads
  sched_mfma_seq<0, S, P, F, L, Wn>();
}

template <int BM, int BN, int WM, int WN, bool GATED>
__global__ __launch_bounds__(WM* WN* kWave) __attribute__((amdgpu_waves_per_eu(1, 1))) void tiled_kernel(
    GemmArgs a) {
  constexpr int kThreads = WM * WN * kWave;
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  constexpr int X_CH = BM * 8 / kThreads;
  constexpr int W_CH = BN * 8 / kThreads;
  constexpr int RSTRIDE = kThreads / 8;  // rows between a thread's consecutive chunks
  constexpr int kXBytes = BM * 128;
  constexpr int kBufBytes = (BM + BN) * 128;
  constexpr int OUT_COLS = GATED ? BN / 2 : BN;
  static_assert(TM >= 1 && TN >= 1 && (!GATED || TN % 2 == 0), "tile shape");
  static_assert(X_CH * kThreads == BM * 8 && W_CH * kThreads == BN * 8, "chunking");
  static_assert(RSTRIDE % 16 == 0, "swizzle key repeats every 16 rows");

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
  int tile = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
  if (tile >= total_tiles) return;

  const int cc = tid & 7;   // 16-byte chunk of a 128-byte K-block row
  const int r0 = tid >> 3;  // first row this thread stages
  const int x_lds0 = r0 * 128 + ((cc ^ swz(r0)) << 4);
  const int w_lds0 = kXBytes + x_lds0;
  const int frag_slot = swz(lrow);  // swizzle key of the rows a lane reads
  const int nkb = ceil_div(a.K, kBK);
  static_assert(!GATED || (WTN / 2) % RSTRIDE == 0, "gate/up half of a chunk is static");

  struct TileInfo {
    int g, row_base, m, m0, nt;
  };
  auto tile_info = [&](int t) {
    TileInfo ti;
    const int mt = t / n_tiles_n;
    ti.nt = t - mt * n_tiles_n;
    ti.g = 0;
    ti.row_base = 0;
    ti.m = a.static_rows;
    ti.m0 = mt * BM;
    if (a.offsets != nullptr) {
      int lo = 0, hi = a.groups - 1;
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (mt_prefix[mid] <= mt) lo = mid; else hi = mid - 1;
      }
      ti.g = lo;
      ti.row_base = a.offsets[lo];
      ti.m = a.offsets[lo + 1] - ti.row_base;
      ti.m0 = (mt - mt_prefix[lo]) * BM;
    }
    // every field is the same across the workgroup; keep it in scalar registers
    ti.g = __builtin_amdgcn_readfirstlane(ti.g);
    ti.row_base = __builtin_amdgcn_readfirstlane(ti.row_base);
    ti.m = __builtin_amdgcn_readfirstlane(ti.m);
    ti.m0 = __builtin_amdgcn_readfirstlane(ti.m0);
    ti.nt = __builtin_amdgcn_readfirstlane(ti.nt);
    return ti;
  };

  // Buffer loads: the tile's bases live in scalar resource descriptors and
  // each staged chunk keeps one 32-bit byte offset.  Offsets >= 2^31 lie past
  // num_records, so rows past the group, columns past N and the K tail read
  // as zeros without touching memory.
  constexpr uint32_t kInvalid = 0x80000000u;
  constexpr int kRecords = 0x7fffffff;
  constexpr int kRsrcWord3 = 0x00020000;
  __amdgpu_buffer_rsrc_t rs_x, rs_w0, rs_w1;
  uint32_t xoff[X_CH], woff[W_CH];
  auto setup = [&](const TileInfo& ti) {
    rs_x = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(a.x + static_cast<size_t>(ti.row_base + ti.m0) * a.K), 0, kRecords, kRsrcWord3);
    const size_t wg = static_cast<size_t>(ti.g) * a.group_stride;
    const int col0 = ti.nt * OUT_COLS;
    rs_w0 = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(a.w0 + wg + static_cast<size_t>(col0) * a.ldw),
                                              0, kRecords, kRsrcWord3);
    rs_w1 = rs_w0;
    if constexpr (GATED)
      rs_w1 = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(a.w1 + wg + static_cast<size_t>(col0) * a.ldw),
                                                0, kRecords, kRsrcWord3);
#pragma unroll
    for (int i = 0; i < X_CH; ++i) {
      const int r = r0 + i * RSTRIDE;
      xoff[i] = (ti.m0 + r < ti.m) ? static_cast<uint32_t>(r * a.K * 2 + cc * 16) : kInvalid;
    }
#pragma unroll
    for (int i = 0; i < W_CH; ++i) {
      const int n = r0 + i * RSTRIDE;
      int lcol;  // column relative to col0
      if constexpr (GATED) {
        const int wn_ = n / WTN, within = n % WTN;
        lcol = wn_ * (WTN / 2) + within % (WTN / 2);
      } else {
        lcol = n;
      }
      woff[i] = (col0 + lcol < a.N) ? static_cast<uint32_t>(lcol * a.ldw * 2) : kInvalid;
    }
  };

  // staging registers: the next K-block is in flight while this one feeds the MFMAs
  u32x4 sx0[X_CH], sw0[W_CH];
  auto load_block = [&](int kb, u32x4 (&rx)[X_CH], u32x4 (&rw)[W_CH]) {
    // K offsets are added to the per-chunk offsets (each below 2^31, so the
    // sum cannot wrap) and the K-tail mark is or-ed in afterwards
    const int kk = kb * kBK + cc * 8;
    const uint32_t kmask = (kb < nkb && kk < a.K) ? 0u : kInvalid;  // past the end: no traffic
    const uint32_t wk = static_cast<uint32_t>((kk < a.K ? weight_col_offset(a, kk) : 0) * 2);
    const uint32_t xk = static_cast<uint32_t>(kb * kBK * 2);
#pragma unroll
    for (int i = 0; i < X_CH; ++i)
      rx[i] = __builtin_amdgcn_raw_buffer_load_b128(rs_x, (xoff[i] + xk) | kmask, 0, 0);
#pragma unroll
    for (int i = 0; i < W_CH; ++i) {
      // a chunk row r0 + i*RSTRIDE lies in the up half iff i*RSTRIDE does (r0 < RSTRIDE)
      const bool up_half = GATED && ((i * RSTRIDE) % WTN) >= WTN / 2;
      rw[i] = __builtin_amdgcn_raw_buffer_load_b128(up_half ? rs_w1 : rs_w0, (woff[i] + wk) | kmask, 0, 0);
    }
  };
  auto store_block = [&](int buf, const u32x4 (&rx)[X_CH], const u32x4 (&rw)[W_CH]) {
    unsigned char* b = smem + buf * kBufBytes;
#pragma unroll
    for (int i = 0; i < X_CH; ++i) *reinterpret_cast<u32x4*>(b + x_lds0 + i * RSTRIDE * 128) = rx[i];
#pragma unroll
    for (int i = 0; i < W_CH; ++i) *reinterpret_cast<u32x4*>(b + w_lds0 + i * RSTRIDE * 128) = rw[i];
  };

  TileInfo cur = tile_info(tile);
  setup(cur);
  load_block(0, sx0, sw0);
  f32x16 acc[TN][TM];

  auto compute = [&](int buf) {
    const unsigned char* b = smem + buf * kBufBytes;
    // fragments double-buffered across the four 16-wide K-steps: the reads
    // of step s+1 are in flight while step s's MFMAs issue
    bf16x8 wf[2][TN], xf[2][TM];
    auto read_frags = [&](int ks, bf16x8 (&w)[TN], bf16x8 (&x)[TM]) {
      const int slot = ((2 * ks + lhalf) ^ frag_slot) << 4;
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
        w[tn] = as_bf16x8(*reinterpret_cast<const u32x4*>(b + kXBytes + (wn * WTN + tn * 32 + lrow) * 128 + slot));
#pragma unroll
      for (int tm = 0; tm < TM; ++tm)
        x[tm] = as_bf16x8(*reinterpret_cast<const u32x4*>(b + (wm * WTM + tm * 32 + lrow) * 128 + slot));
    };
    read_frags(0, wf[0], xf[0]);
#pragma unroll
    for (int ks = 0; ks < kBK / 16; ++ks) {
      if (ks + 1 < kBK / 16) read_frags(ks + 1, wf[(ks + 1) & 1], xf[(ks + 1) & 1]);
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
#pragma unroll
        for (int tm = 0; tm < TM; ++tm)
          acc[tn][tm] = mfma32x32x16(wf[ks & 1][tn], xf[ks & 1][tm], acc[tn][tm]);
    }
  };
  // One K-block, a single basic block so the scheduler can interleave it:
  // load block kb+1 into registers, multiply block kb from LDS, store kb+1
  // into the other LDS buffer (past the last block the loads are masked and
  // the store lands in the idle buffer).
  auto kblock = [&](int kb) {
    load_block(kb + 1, sx0, sw0);
    compute(kb & 1);
    store_block((kb + 1) & 1, sx0, sw0);
    sched_kblock<kBK / 16, TM * TN, TM + TN, X_CH + W_CH, X_CH + W_CH>();
    __syncthreads();
  };

  while (true) {
    store_block(0, sx0, sw0);
    __syncthreads();
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
#pragma unroll
      for (int tm = 0; tm < TM; ++tm) acc[tn][tm] = f32x16{};
    for (int kb = 0; kb < nkb; ++kb) kblock(kb);

    // start the next tile's first K-block before this tile's epilogue
    const int next = tile + gridDim.x;
    TileInfo nxt{};
    if (next < total_tiles) {
      nxt = tile_info(next);
      setup(nxt);
      load_block(0, sx0, sw0);
    }

    // epilogue: lane holds C[n = 8*(v/4) + 4*lhalf + v%4][t = lrow] per 32x32 tile
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) {
      const int row = cur.m0 + wm * WTM + tm * 32 + lrow;
      if (row >= cur.m) continue;
      uint16_t* orow = a.out + static_cast<size_t>(cur.row_base + row) * a.N;
      constexpr int TOUT = GATED ? TN / 2 : TN;
#pragma unroll
      for (int tn = 0; tn < TOUT; ++tn) {
#pragma unroll
        for (int v4 = 0; v4 < 4; ++v4) {
          const int col = GATED ? cur.nt * OUT_COLS + wn * (WTN / 2) + tn * 32 + 8 * v4 + 4 * lhalf
                                : cur.nt * BN + wn * WTN + tn * 32 + 8 * v4 + 4 * lhalf;
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
    if (next >= total_tiles) break;
    tile = next;
    cur = nxt;
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
  constexpr int kWgsPerCu = static_cast<int>((160 * 1024) / (kLds + 8 * 1024)) > 0
                                ? static_cast<int>((160 * 1024) / (kLds + 8 * 1024))
                                : 1;
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
  long long grid = std::min<long long>(tiles, static_cast<long long>(device_cu_count()) * kWgsPerCu);
  grid = ((grid + 7) / 8) * 8;
  hipLaunchKernelGGL((tiled_kernel<BM, BN, WM, WN, GATED>), dim3(static_cast<unsigned>(grid)),
                     dim3(kThreads), kLds, st, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_tiled(const Segments& seg, const GemmArgs& a, bool gated, hipStream_t st) {
  if (seg.groups > kMaxGroups) return hipErrorInvalidValue;
  return gated ? launch_tiled_t<256, 256, 4, 2, true>(seg, a, st)
               : launch_tiled_t<256, 256, 4, 2, false>(seg, a, st);
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
