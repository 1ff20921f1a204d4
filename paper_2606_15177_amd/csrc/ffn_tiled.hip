// Expert FFN for prefill-sized batches: a persistent bf16 MFMA grouped GEMM
// with direct-to-LDS loads and two ping-pong wave groups.
//
// Tiles.  An output tile is 256 token rows x 256 weight rows of one group
// (expert).  For the gate/up GEMM the 256 weight rows are 128 gate rows and
// the 128 up rows of the same output columns, so a tile yields 128 columns of
// h = silu(gate) * up.  The tile list is implied by the device-side offsets:
// every workgroup computes the per-group prefix of ceil(rows/256) once, then
// walks tile ids t, t+gridDim, ... where t renumbers workgroups so that each
// XCD (workgroups are dealt round-robin to the 8 XCDs) owns a contiguous run
// of tiles.  Tiles are numbered group-major, then by n-tile, then by m-tile,
// so the m-tiles that share a weight tile run side by side on one XCD and
// the weights are fetched from HBM once.  Group sizes never leave the
// device.
//
// Stages.  K advances in stages of 32.  A stage holds X[256 x 32] and
// W[256 x 32] in LDS (64-byte rows, 32 KB) and is filled by
// buffer_load_dwordx4 ... lds, which writes 64 lanes x 16 bytes to
// consecutive LDS addresses without passing through registers.  Four stages
// form a ring: the loads of stage j+3 are issued while stage j is consumed,
// so a load has about three stage times to arrive, and the stage sequence
// runs on across tile boundaries (the next tile's first stages are in flight
// during a tile's last ones).  Chunk c (16 bytes) of LDS row r sits at slot
// c ^ ((r >> 2) & 3): every lane of a load fetches the global chunk that
// belongs at its fixed LDS slot, and the 16 rows that 16 lanes of an MFMA
// fragment read land in 16 distinct bank groups.  Rows past a group's end,
// columns past N and the K tail get byte offsets >= 2^31, past the buffer
// descriptor's range: they read as zeros and cost no memory traffic.
//
// Ping-pong.  The 8 waves form two groups of four, one wave of each group
// per SIMD.  Group 0 computes token rows 0..127 of the tile and group 1 rows
// 128..255; a wave owns 64 token rows x 128 weight rows (2 x 4 MFMA tiles of
// v_mfma_f32_32x32x16_bf16, weights as the A operand, tokens as B).  The two
// groups alternate, one phase apart, between a memory phase (issue loads,
// read the stage's fragments from LDS into registers) and a compute phase
// (16 MFMAs on registers only), with a workgroup barrier between phases: on
// every SIMD one wave issues MFMAs while the other one feeds LDS.
//
// Waits.  Each wave issues the loads of stage j+3 for its part in its memory
// phase of stage j and waits for its own loads of stage j+1 (s_waitcnt vmcnt
// with the two younger stages' 8 loads still in flight) before the barrier
// that precedes the first read of stage j+1; it waits for its LDS reads
// (lgkmcnt(0)) before every barrier, so a buffer is refilled only after both
// groups have read it.
#include "ffn_impl.h"

namespace moe {
namespace {

constexpr int kBM = 256;                          // token rows per tile
constexpr int kBN = 256;                          // weight rows per tile
constexpr int kBK = 32;                           // K per stage
constexpr int kStages = 4;                        // LDS ring depth
constexpr int kThreads = 8 * kWave;
constexpr int kRowBytes = kBK * 2;                // 64
constexpr int kPartBytes = kBM * kRowBytes;       // one operand of a stage: 16 KB
constexpr int kStageBytes = 2 * kPartBytes;       // X part, then W part
constexpr int kLdsBytes = kStages * kStageBytes;  // 128 KB
constexpr int kLoadsPerStage = 4;                 // per wave: 4 loads of 1 KB (group 0: X, group 1: W)
constexpr int kMaxGroups = 1024;
static_assert(kBM == kBN && kBM * kRowBytes == 16 * 1024 * 1, "a stage part is 16 loads of 1 KB");

// s_waitcnt immediates (gfx9 layout: vmcnt [3:0] and [15:14], expcnt [6:4],
// lgkmcnt [11:8]); a field at its maximum does not wait.
constexpr int wait_vm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }
constexpr int kWaitLgkm0 = 15 | (3 << 14) | (7 << 4);
constexpr int kWaitAll = 0;

// Workgroup barrier that also fences the compiler: no instruction is moved
// across it, and memory accesses stay on their side (the hardware waits are
// the explicit s_waitcnt above).
__device__ __forceinline__ void phase_barrier() {
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("s_barrier" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
}

// 64 lanes x 16 bytes from rsrc + voff[lane] to lds + 16 * lane.
__device__ __forceinline__ void load_lds16(__amdgpu_buffer_rsrc_t rs, unsigned char* lds, uint32_t voff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (__attribute__((address_space(3))) void*)lds, 16, voff, 0, 0, 0);
}

template <bool GATED>
__global__ __launch_bounds__(kThreads) void tiled_kernel(GemmArgs a) {
  constexpr int OUT_COLS = GATED ? kBN / 2 : kBN;
  constexpr uint32_t kInvalid = 0x80000000u;
  constexpr int kRecords = 0x7fffffff;
  constexpr int kRsrcWord3 = 0x00020000;

  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  __shared__ int mt_prefix[kMaxGroups + 1];  // first m-tile of each group
  __shared__ int row_off[kMaxGroups + 1];    // the group offsets, read once

  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int grp = wave >> 2, q = wave & 3;
  const int lrow = lane & 31, lhalf = lane >> 5;
  const int n_tiles_n = ceil_div(a.N, OUT_COLS);

  int total_mt;
  if (a.offsets == nullptr) {
    total_mt = ceil_div(a.static_rows, kBM);
  } else {
    if (wave == 0) {
      int carry = 0;
      for (int g0 = 0; g0 < a.groups; g0 += kWave) {
        const int g = g0 + lane;
        int cnt = 0;
        if (g < a.groups) {
          const int lo = a.offsets[g], hi = a.offsets[g + 1];
          row_off[g] = lo;
          if (g + 1 == a.groups) row_off[g + 1] = hi;
          cnt = ceil_div(hi - lo, kBM);
        }
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
  const int first = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
  if (first >= total_tiles) return;
  const int nkb = ceil_div(a.K, kBK);
  const int n_stages = ceil_div(total_tiles - first, gridDim.x) * nkb;

  struct TileInfo {
    int g, row_base, m, m0, nt;
  };
  // Tile order: group, then n-tile, then m-tile (fastest).  The m-tiles of a
  // group that share one weight tile are neighbours, so they run at the same
  // time on one XCD and the weights cross the fabric once.
  auto tile_info = [&](int t) {
    TileInfo ti;
    int mg = total_mt, base = 0;  // m-tiles of the group, first tile id of the group
    ti.g = 0;
    ti.row_base = 0;
    ti.m = a.static_rows;
    if (a.offsets != nullptr) {
      int lo = 0, hi = a.groups - 1;
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (mt_prefix[mid] * n_tiles_n <= t) lo = mid; else hi = mid - 1;
      }
      // from LDS: a global load here would make the compiler wait for every
      // stage load in flight (they share the vector memory counter)
      ti.g = lo;
      ti.row_base = row_off[lo];
      ti.m = row_off[lo + 1] - ti.row_base;
      base = mt_prefix[lo] * n_tiles_n;
      mg = mt_prefix[lo + 1] - mt_prefix[lo];
    }
    const int local = t - base;
    ti.nt = local / mg;
    ti.m0 = (local - ti.nt * mg) * kBM;
    ti.g = __builtin_amdgcn_readfirstlane(ti.g);
    ti.row_base = __builtin_amdgcn_readfirstlane(ti.row_base);
    ti.m = __builtin_amdgcn_readfirstlane(ti.m);
    ti.m0 = __builtin_amdgcn_readfirstlane(ti.m0);
    ti.nt = __builtin_amdgcn_readfirstlane(ti.nt);
    return ti;
  };

  // ---- load side: runs three stages ahead of the compute side ----
  // Group 0 fills the X part of every stage and group 1 the W part, each in
  // its own memory phase, so no wave issues loads between its MFMAs.  Wave q
  // of a group fills the 16-row blocks 4q..4q+3 of its part.  A lane's LDS
  // slot is lane & 3 of row lane >> 2 of a block, so the global chunk it
  // fetches, (lane & 3) ^ ((row >> 2) & 3), depends on the lane only.
  const int chunk = (lane & 3) ^ ((lane >> 4) & 3);
  __amdgpu_buffer_rsrc_t rs_ld;  // X (group 0) or W (group 1) of the tile being loaded
  u32x4 ld_off;                  // byte offset of each load's row, or >= 2^31
  int ld_tile = first, ld_kb = 0;
  auto ld_setup = [&](int t) {
    if (t >= total_tiles) {  // past this workgroup's last tile: empty loads keep the count regular
      ld_off = u32x4{kInvalid, kInvalid, kInvalid, kInvalid};
      return;
    }
    const TileInfo ti = tile_info(t);
    if (grp == 0) {
      // token rows: consecutive rows of x, or x rows named by x_rows (the
      // dispatch gather done by the loads themselves)
      const uint16_t* xb = a.x_rows ? a.x : a.x + static_cast<size_t>(ti.row_base + ti.m0) * a.K;
      rs_ld = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(xb), 0, kRecords, kRsrcWord3);
      // the four row indices are loaded together (rows past the group read
      // the group's first index and are masked), so one wait covers them
      int xr[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = 16 * (4 * q + i) + (lane >> 2);  // token row within the tile
        xr[i] = r;
        if (a.x_rows) xr[i] = a.x_rows[ti.row_base + (ti.m0 + r < ti.m ? ti.m0 + r : 0)];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = 16 * (4 * q + i) + (lane >> 2);
        ld_off[i] = ti.m0 + r < ti.m ? static_cast<uint32_t>(xr[i] * a.K * 2 + chunk * 16) : kInvalid;
      }
    } else {
      const int col0 = ti.nt * OUT_COLS;
      // the wave's 64 weight rows 64q..64q+63 are all gate rows or all up rows
      const bool up = GATED && (q & 1);
      const uint16_t* wbase = (up ? a.w1 : a.w0) + static_cast<size_t>(ti.g) * a.group_stride +
                              static_cast<size_t>(col0) * a.ldw;
      rs_ld = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(wbase), 0, kRecords, kRsrcWord3);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = 16 * (4 * q + i) + (lane >> 2);            // weight row within the tile
        const int lcol = GATED ? (r >> 7) * 64 + (r & 63) : r;  // output column relative to col0
        ld_off[i] = (col0 + lcol < a.N) ? static_cast<uint32_t>(lcol * a.ldw * 2 + chunk * 16) : kInvalid;
      }
    }
  };
  // Byte offset of the stage's K origin (added to every load's row-and-chunk
  // offset) and the mark of a chunk past K.  The offset is the same for all
  // lanes except for weights whose K range is stacked from segments that a
  // 32-wide stage can straddle.
  uint32_t ld_k = 0, ld_kmask = 0;
  auto ld_kstep = [&]() {
    const int k0 = ld_kb * kBK;
    ld_kmask = k0 + chunk * 8 < a.K ? 0u : kInvalid;
    if (grp == 0 || a.kseg >= a.K) {
      ld_k = static_cast<uint32_t>(k0 * 2);
    } else if (a.kseg % kBK == 0) {
      const int seg = k0 / a.kseg;
      ld_k = static_cast<uint32_t>((static_cast<size_t>(seg) * a.seg_stride + (k0 - seg * a.kseg)) * 2);
    } else {
      const int kk = min(k0 + chunk * 8, a.K - 8);
      ld_k = static_cast<uint32_t>((weight_col_offset(a, kk) - static_cast<size_t>(kk - k0)) * 2);
    }
  };
  // load i (of 4) of this wave's part of the stage being loaded, into buffer buf
  auto load_one = [&](int buf, int i) {
    load_lds16(rs_ld, smem + buf * kStageBytes + grp * kPartBytes + q * 4096 + i * 1024,
               (ld_off[i] + ld_k) | ld_kmask);
  };
  auto ld_advance = [&]() {  // after the four loads of a stage
    if (++ld_kb == nkb) {
      ld_kb = 0;
      ld_tile += gridDim.x;
      ld_setup(ld_tile);
    }
    ld_kstep();
  };
  auto issue = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 4; ++i) load_one(buf, i);
    ld_advance();
  };

  // ---- compute side ----
  const int xrow0 = grp * 128 + (q & 1) * 64;  // this wave's token rows in the tile
  const int wrow0 = (q >> 1) * 128;            // and its weight rows
  const int rsw = (lrow >> 2) & 3;             // slot key of the rows this lane reads
  bf16x8 xf[2][2], wf[2][4];                   // [k-step][tile]
  f32x16 acc[4][2];
  auto read_frags = [&](int buf, int ks) {  // the fragments of one K-step
    const unsigned char* b = smem + buf * kStageBytes;
    {
      const int slot = ((2 * ks + lhalf) ^ rsw) << 4;
#pragma unroll
      for (int tn = 0; tn < 4; ++tn)
        wf[ks][tn] = as_bf16x8(*reinterpret_cast<const u32x4*>(b + kPartBytes + (wrow0 + tn * 32 + lrow) * kRowBytes + slot));
#pragma unroll
      for (int tm = 0; tm < 2; ++tm)
        xf[ks][tm] = as_bf16x8(*reinterpret_cast<const u32x4*>(b + (xrow0 + tm * 32 + lrow) * kRowBytes + slot));
    }
  };
  auto mfma_step = [&](int ks) {
#pragma unroll
    for (int tn = 0; tn < 4; ++tn)
#pragma unroll
      for (int tm = 0; tm < 2; ++tm) acc[tn][tm] = mfma32x32x16(wf[ks][tn], xf[ks][tm], acc[tn][tm]);
  };
  auto zero_acc = [&]() {
#pragma unroll
    for (int tn = 0; tn < 4; ++tn)
#pragma unroll
      for (int tm = 0; tm < 2; ++tm) acc[tn][tm] = f32x16{};
  };
  // lane holds C[n = 8*(v/4) + 4*lhalf + v%4][t = lrow] of each 32x32 tile
  auto epilogue = [&](const TileInfo& ti) {
#pragma unroll
    for (int tm = 0; tm < 2; ++tm) {
      const int row = ti.m0 + xrow0 + tm * 32 + lrow;
      if (row >= ti.m) continue;
      uint16_t* orow = a.out + static_cast<size_t>(ti.row_base + row) * a.N;
      constexpr int TOUT = GATED ? 2 : 4;
#pragma unroll
      for (int tn = 0; tn < TOUT; ++tn) {
#pragma unroll
        for (int v4 = 0; v4 < 4; ++v4) {
          const int col = ti.nt * OUT_COLS + (q >> 1) * (GATED ? 64 : 128) + tn * 32 + 8 * v4 + 4 * lhalf;
          if (col >= a.N) continue;
          float o[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float c0 = acc[tn][tm][4 * v4 + i];
            if constexpr (GATED)
              o[i] = silu(c0) * acc[tn + 2][tm][4 * v4 + i];
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
  };

  // ---- pipeline ----
  TileInfo cur = tile_info(first);
  int cur_tile = first, kb = 0;
  zero_acc();
  ld_setup(first);
  ld_kstep();
  issue(0);
  issue(1);
  issue(2);
  __builtin_amdgcn_s_waitcnt(wait_vm(2 * kLoadsPerStage));  // own stage-0 loads landed
  phase_barrier();
  if (grp == 1) phase_barrier();  // group 1 runs one phase behind
  for (int j = 0; j < n_stages; ++j) {
    // memory phase of stage j
    if (kb == 0 && j > 0) {
      epilogue(cur);
      zero_acc();
      cur_tile += gridDim.x;
      cur = tile_info(cur_tile);
    }
    // The stage's four loads are spread over both phases, between the LDS
    // reads and between the MFMAs: the texture unit takes them one by one
    // and no wave stalls on a burst of loads.
    const int lb = (j + 3) & 3;
    load_one(lb, 0);
    read_frags(j & 3, 0);
    load_one(lb, 1);
    read_frags(j & 3, 1);
    __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 6, 0);
    __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 6, 0);
    if (grp == 1) __builtin_amdgcn_s_waitcnt(wait_vm(kLoadsPerStage + 2));  // own stage j+1 landed
    __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
    phase_barrier();
    // compute phase of stage j
    mfma_step(0);
    load_one(lb, 2);
    mfma_step(1);
    load_one(lb, 3);
    __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
    __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
    __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
    if (grp == 0) __builtin_amdgcn_s_waitcnt(wait_vm(2 * kLoadsPerStage));  // own stage j+1 landed
    phase_barrier();
    ld_advance();
    if (++kb == nkb) kb = 0;
  }
  if (grp == 0) phase_barrier();  // matches group 1's extra barrier
  epilogue(cur);
  __builtin_amdgcn_s_waitcnt(kWaitAll);  // no load may land in LDS after the workgroup ends
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

template <bool GATED>
hipError_t launch_tiled_t(const Segments& seg, const GemmArgs& a, hipStream_t st) {
  constexpr int OUT_COLS = GATED ? kBN / 2 : kBN;
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&tiled_kernel<GATED>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, kLdsBytes);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  const long long m_tiles = (a.offsets ? static_cast<long long>(ceil_div(seg.total_rows, kBM)) + seg.groups
                                       : ceil_div(seg.static_rows, kBM));
  const long long tiles = m_tiles * ceil_div(a.N, OUT_COLS);
  if (tiles == 0) return hipSuccess;
  long long grid = std::min<long long>(tiles, device_cu_count());  // one workgroup per CU (LDS)
  grid = ((grid + 7) / 8) * 8;
  hipLaunchKernelGGL((tiled_kernel<GATED>), dim3(static_cast<unsigned>(grid)), dim3(kThreads), kLdsBytes, st, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_tiled(const Segments& seg, const GemmArgs& a, bool gated, hipStream_t st) {
  if (seg.groups > kMaxGroups || a.x_blocked || a.out_blocked) return hipErrorInvalidValue;
  // 32-bit byte offsets: a tile's X rows (all of x when rows are indexed) and
  // a group's weight columns
  const size_t x_span = static_cast<size_t>(a.x_rows ? a.x_row_count : kBM) * a.K * 2;
  const size_t w_span = (static_cast<size_t>(kBN) * a.ldw +
                         (a.kseg < a.K ? static_cast<size_t>((a.K - 1) / a.kseg) * a.seg_stride : 0) + a.K) * 2;
  if (x_span >= 0x80000000ull || w_span >= 0x80000000ull) return hipErrorInvalidValue;
  return gated ? launch_tiled_t<true>(seg, a, st) : launch_tiled_t<false>(seg, a, st);
}

bool ffn_streams_weights(const Segments& seg) { return seg.max_rows <= kSkinnyMaxRows; }

hipError_t launch_ffn_up(const Segments& seg, const UpArgs& u, hipStream_t st) {
  if (u.h_blocked && !ffn_streams_weights(seg)) return hipErrorInvalidValue;
  if (u.x_rows && (seg.offsets == nullptr || u.x_row_count <= 0)) return hipErrorInvalidValue;
  GemmArgs a{};
  a.x = u.x;
  a.x_rows = u.x_rows;
  a.x_row_count = u.x_row_count;
  a.out_blocked = u.h_blocked;
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
  if (d.h_blocked && !ffn_streams_weights(seg)) return hipErrorInvalidValue;
  GemmArgs a{};
  a.x = d.h;
  a.x_blocked = d.h_blocked;
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
