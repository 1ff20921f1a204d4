// Expert FFN for prefill-sized batches: a persistent bf16 MFMA grouped GEMM
// with direct-to-LDS loads, one wave per SIMD.
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
// Waves.  Four waves, one per SIMD; wave (wm, wn) owns token rows
// 128*wm .. +127 and weight rows 128*wn .. +127 of the tile: 4 x 4
// v_mfma_f32_32x32x16_bf16 tiles (weights as the A operand, tokens as B),
// 256 fp32 accumulators held in AGPRs.
//
// Stages.  K advances in stages of 32.  A stage holds X[256 x 32] and
// W[256 x 32] in LDS (64-byte rows, 32 KB) and is filled by
// buffer_load_dwordx4 ... lds, which writes 64 lanes x 16 bytes to
// consecutive LDS addresses without passing through registers; each wave
// fills 64 rows of each part.  Four stages form a ring.  Chunk c (16 bytes)
// of LDS row r sits at slot c ^ ((r >> 2) & 3): every lane of a load fetches
// the global chunk that belongs at its fixed LDS slot, and the 16 rows that
// 16 lanes of an MFMA fragment read land in 16 distinct bank groups.  Rows
// past a group's end, columns past N and the K tail get byte offsets
// >= 2^31, past the buffer descriptor's range: they read as zeros and cost
// no memory traffic.
//
// Pipeline.  One workgroup barrier per stage, placed before its last K-step
// after each wave has waited for its own loads of the next stage and for its
// LDS reads: past it the next stage's data are in LDS and the stage's own
// buffer is free.  The loads of stage j + 4 go into that buffer, spread one
// per four MFMAs over the last K-step of stage j and the first of stage
// j + 1: a burst of loads stalls the issuing wave (one wave per SIMD, in
// order) while the address unit drains, and the MFMA pipe with it.  A load
// has about three stage times to land; the stage sequence runs on across
// tile boundaries.
//
// Epilogue.  A lane holds row r, columns 8*v + 4*h + 0..3 (v < 4, h = lane
// half) of each 32 x 32 accumulator tile.  Values are converted in bf16
// pairs and a swap between the lane halves (v_permlane32_swap) gives every
// lane 8 consecutive columns, written as one 16-byte store.
#include "ffn_impl.h"

namespace moe {
namespace {

constexpr int kBM = 256;                // token rows per tile
constexpr int kBN = 256;                // weight rows per tile
constexpr int kThreads = 4 * kWave;     // four waves, one per SIMD
constexpr int kMaxGroups = 1024;

// One K stage and the ring of them.
struct Stage {
  static constexpr int BK = 32;                   // K per stage
  static constexpr int CPR = BK * 2 / 16;         // 16-byte chunks per LDS row
  static constexpr int RPI = kWave / CPR;         // rows per load instruction
  static constexpr int SWZ = 16 / CPR;            // rows sharing one swizzle key
  static constexpr int ROW = BK * 2;              // bytes per LDS row
  static constexpr int PART = kBM * ROW;          // one operand of a stage: 16 KB
  static constexpr int STAGE = 2 * PART;          // X part, then W part
  static constexpr int NS = 4;                    // ring depth
  static constexpr int LDS = NS * STAGE;          // 128 KB
  static constexpr int LPP = 64 / RPI;            // loads per part per wave
  static constexpr int LPS = 2 * LPP;             // loads per stage per wave
  static constexpr int KSTEPS = BK / 16;          // MFMA K-steps per stage
};
static_assert(kBM == kBN && Stage::RPI * Stage::ROW == 1024, "a load fills 1 KB of LDS rows");

// s_waitcnt immediates (gfx9 layout: vmcnt [3:0] and [15:14], expcnt [6:4],
// lgkmcnt [11:8]); a field at its maximum does not wait.
constexpr int wait_vm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }
constexpr int kWaitLgkm0 = 15 | (3 << 14) | (7 << 4);
constexpr int kWaitAll = 0;

// Workgroup barrier that also fences the compiler: no instruction is moved
// across it, and memory accesses stay on their side (the hardware waits are
// the explicit s_waitcnt).
__device__ __forceinline__ void phase_barrier() {
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("s_barrier" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
}

// 64 lanes x 16 bytes from rsrc + voff[lane] to lds + 16 * lane.
__device__ __forceinline__ void load_lds16(__amdgpu_buffer_rsrc_t rs, unsigned char* lds, uint32_t voff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (__attribute__((address_space(3))) void*)lds, 16, voff, 0, 0, 0);
}

// The lane id, recomputed behind a volatile asm: values derived from it are
// not hoisted out of loops by the compiler and hold no register across them.
__device__ __forceinline__ int opaque_lane_id() {
  int ln;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(ln));
  return ln;
}

template <bool GATED>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(1, 1))) void tiled_kernel(GemmArgs a) {
  using C = Stage;
  constexpr int OUT_COLS = GATED ? kBN / 2 : kBN;
  constexpr uint32_t kInvalid = 0x80000000u;
  constexpr int kRecords = 0x7fffffff;
  constexpr int kRsrcWord3 = 0x00020000;

  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  __shared__ int mt_prefix[kMaxGroups + 1];
  __shared__ int row_off[kMaxGroups + 1];

  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int wm = wave & 1, wn = wave >> 1;
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
  const int per_xcd = gridDim.x / 8;
  const int first = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
  if (first >= total_tiles) return;
  const int nkb = ceil_div(a.K, C::BK);
  const int n_stages = ceil_div(total_tiles - first, gridDim.x) * nkb;

  struct TileInfo {
    int g, row_base, m, m0, nt;
  };
  auto tile_info = [&](int t) {
    TileInfo ti;
    int mg = total_mt, base = 0;
    ti.g = 0;
    ti.row_base = 0;
    ti.m = a.static_rows;
    if (a.offsets != nullptr) {
      int lo = 0, hi = a.groups - 1;
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (mt_prefix[mid] * n_tiles_n <= t) lo = mid; else hi = mid - 1;
      }
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

  // ---- load side: wave w fills rows 64w..64w+63 of both parts ----
  // Load i writes rows 64w + RPI*i + lane/CPR, slot lane%CPR; the global
  // chunk it fetches is slot ^ ((row / SWZ) % CPR).
  const int lslot = lane % C::CPR;
  __amdgpu_buffer_rsrc_t rs_x, rs_w0, rs_w1;
  uint32_t xoff[C::LPP], woff[C::LPP];
  int ld_tile = first, ld_kb = 0;
  auto ld_chunk_l = [&](int i, int ln) {
    const int r = 64 * wave + C::RPI * i + ln / C::CPR;
    return (ln % C::CPR) ^ ((r / C::SWZ) % C::CPR);
  };
  auto ld_chunk = [&](int i) { return ld_chunk_l(i, lane); };
  auto ld_setup = [&](int t_in) {
    // past this workgroup's last tile: the same loads with every offset
    // marked invalid keep the load count regular (branch-free, so the
    // offsets stay in registers)
    const bool live = t_in < total_tiles;
    const uint32_t dead = live ? 0u : kInvalid;
    const int t = live ? t_in : total_tiles - 1;
    const TileInfo ti = tile_info(t);
    // opaque lane id: the per-lane row terms are recomputed here rather
    // than hoisted out of the K loop
    int ln = opaque_lane_id();
    const uint16_t* xb = a.x_rows ? a.x : a.x + static_cast<size_t>(ti.row_base + ti.m0) * a.K;
    rs_x = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(xb), 0, kRecords, kRsrcWord3);
    int xr[C::LPP];
#pragma unroll
    for (int i = 0; i < C::LPP; ++i) {
      const int r = 64 * wave + C::RPI * i + ln / C::CPR;
      xr[i] = r;
      if (a.x_rows) xr[i] = a.x_rows[ti.row_base + (ti.m0 + r < ti.m ? ti.m0 + r : 0)];
    }
#pragma unroll
    for (int i = 0; i < C::LPP; ++i) {
      const int r = 64 * wave + C::RPI * i + ln / C::CPR;
      xoff[i] = (ti.m0 + r < ti.m ? static_cast<uint32_t>(xr[i] * a.K * 2 + ld_chunk_l(i, ln) * 16) : kInvalid) | dead;
    }
    const int col0 = ti.nt * OUT_COLS;
    const size_t gofs = static_cast<size_t>(ti.g) * a.group_stride + static_cast<size_t>(col0) * a.ldw;
    rs_w0 = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(a.w0 + gofs), 0, kRecords, kRsrcWord3);
    if (GATED) rs_w1 = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(a.w1 + gofs), 0, kRecords, kRsrcWord3);
#pragma unroll
    for (int i = 0; i < C::LPP; ++i) {
      const int r = 64 * wave + C::RPI * i + ln / C::CPR;  // weight row of the tile
      const int lcol = GATED ? (r >> 7) * 64 + (r & 63) : r;
      woff[i] = ((col0 + lcol < a.N) ? static_cast<uint32_t>(lcol * a.ldw * 2 + ld_chunk_l(i, ln) * 16) : kInvalid) | dead;
    }
  };
  // the 64 weight rows of this wave are all gate rows or all up rows
  const bool w_up = GATED && (wave & 1);
  // Per stage and lane: the K offset of X and of W and the past-K mark for
  // the (at most two) chunks a lane fetches; p = load index parity.
  uint32_t kx0 = 0, kx1 = 0, kw0 = 0, kw1 = 0;
  auto kstep_one = [&](int p, uint32_t& kx, uint32_t& kw) {
    const int k0 = ld_kb * C::BK;
    const int ch = ld_chunk(p);
    const uint32_t mask = k0 + ch * 8 < a.K ? 0u : kInvalid;
    kx = static_cast<uint32_t>(k0 * 2) | mask;
    uint32_t w;
    if (a.kseg >= a.K) {
      w = static_cast<uint32_t>(k0 * 2);
    } else if (a.kseg % C::BK == 0) {
      const int seg = k0 / a.kseg;
      w = static_cast<uint32_t>((static_cast<size_t>(seg) * a.seg_stride + (k0 - seg * a.kseg)) * 2);
    } else {
      const int kk = min(k0 + ch * 8, a.K - 8);
      w = static_cast<uint32_t>((weight_col_offset(a, kk) - static_cast<size_t>(kk - k0)) * 2);
    }
    kw = w | mask;
  };
  auto ld_kstep = [&]() {
    kstep_one(0, kx0, kw0);
    kstep_one(1, kx1, kw1);
  };
  // load l (0..LPS-1) of the stage being loaded into buffer buf: X loads first, then W
  auto load_one = [&](int buf, int l) {
    unsigned char* base = smem + buf * C::STAGE;
    if (l < C::LPP) {
      const uint32_t k = (l & 1) ? kx1 : kx0;
      load_lds16(rs_x, base + wave * (64 * C::ROW) + l * 1024, (xoff[l] + k) | (k & kInvalid));
    } else {
      const int i = l - C::LPP;
      const uint32_t k = (i & 1) ? kw1 : kw0;
      load_lds16(w_up ? rs_w1 : rs_w0, base + C::PART + wave * (64 * C::ROW) + i * 1024,
                 (woff[i] + k) | (k & kInvalid));
    }
  };
  auto ld_advance = [&]() {
    if (++ld_kb == nkb) {
      ld_kb = 0;
      ld_tile += gridDim.x;
      ld_setup(ld_tile);
    }
    ld_kstep();
  };

  // ---- compute side: token rows 128wm.., weight rows 128wn.. ----
  const int xrow0 = wm * 128, wrow0 = wn * 128;
  const int rsw = (lrow / C::SWZ) % C::CPR;
  bf16x8 xf[2][4], wf[2][4];
  f32x16 acc[4][4];
  auto read_frags = [&](int buf, int ks, int set) {
    const unsigned char* b = smem + buf * C::STAGE;
    const int slot = ((2 * ks + lhalf) ^ rsw) << 4;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      wf[set][t] = as_bf16x8(*reinterpret_cast<const u32x4*>(b + C::PART + (wrow0 + t * 32 + lrow) * C::ROW + slot));
      xf[set][t] = as_bf16x8(*reinterpret_cast<const u32x4*>(b + (xrow0 + t * 32 + lrow) * C::ROW + slot));
    }
  };
  auto mfma_set = [&](int set) {
#pragma unroll
    for (int tn = 0; tn < 4; ++tn)
#pragma unroll
      for (int tm = 0; tm < 4; ++tm) acc[tn][tm] = mfma32x32x16(wf[set][tn], xf[set][tm], acc[tn][tm]);
  };
  auto zero_acc = [&]() {
#pragma unroll
    for (int tn = 0; tn < 4; ++tn)
#pragma unroll
      for (int tm = 0; tm < 4; ++tm) acc[tn][tm] = f32x16{};
  };
  // Lane (erow, ehalf) of a 32x32 accumulator tile holds row erow, columns
  // 8*v4 + 4*ehalf + 0..3.  Values go out in bf16 pairs; a swap between the
  // lane halves gives every lane 8 consecutive columns, one 16-byte store.
  auto epilogue = [&](const TileInfo& ti) {
    // an opaque copy of the lane id keeps the compiler from hoisting the
    // epilogue's per-lane addresses out of the K loop (they would hold
    // registers through it)
    int ln = opaque_lane_id();
    const int erow = ln & 31, ehalf = ln >> 5;
    constexpr int WCOLS = GATED ? 64 : 128;  // output columns of this wave
    const int col_w = ti.nt * OUT_COLS + wn * WCOLS;
    const bool cols_full = col_w + WCOLS <= a.N;
#pragma unroll
    for (int tm = 0; tm < 4; ++tm) {
      const int row = ti.m0 + xrow0 + tm * 32 + erow;
      const bool row_ok = row < ti.m;
      uint16_t* orow = a.out + static_cast<size_t>(ti.row_base + (row_ok ? row : 0)) * a.N;
      constexpr int TOUT = GATED ? 2 : 4;
#pragma unroll
      for (int tn = 0; tn < TOUT; ++tn) {
        uint32_t pk[8];  // pk[2*v4 + h]: columns 8*v4 + 4*ehalf + 2h, +1
#pragma unroll
        for (int v4 = 0; v4 < 4; ++v4) {
          float o[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float c0 = acc[tn][tm][4 * v4 + i];
            if constexpr (GATED)
              o[i] = silu(c0) * acc[tn + 2][tm][4 * v4 + i];
            else
              o[i] = c0;
          }
          pk[2 * v4] = cvt_pk_bf16(o[0], o[1]);
          pk[2 * v4 + 1] = cvt_pk_bf16(o[2], o[3]);
        }
#pragma unroll
        for (int q = 0; q < 2; ++q) {  // columns 16q .. 16q+15 of the 32-column tile
          // lower lanes keep columns 16q+0..3 and take 16q+4..7 from the upper
          // half; upper lanes take 16q+8..11 and keep 16q+12..15
          const auto s0 = __builtin_amdgcn_permlane32_swap(pk[4 * q], pk[4 * q + 2], false, false);
          const auto s1 = __builtin_amdgcn_permlane32_swap(pk[4 * q + 1], pk[4 * q + 3], false, false);
          const u32x4 v = {s0[0], s1[0], s0[1], s1[1]};
          const int col = col_w + tn * 32 + 16 * q + 8 * ehalf;
          if (row_ok && (cols_full || col < a.N)) *reinterpret_cast<u32x4*>(orow + col) = v;
        }
      }
    }
  };

  // ---- pipeline ----
  // The barrier of stage j sits before its last K-step, after every wave's
  // last LDS read of stage j: from then on stage j's buffer takes the loads
  // of stage j + NS.  Their first half is issued among the MFMAs of stage
  // j's last K-step, the second half among those of stage j + 1's first
  // K-step, one load per four MFMAs: a burst of loads stalls the issuing wave
  // (one wave per SIMD) while the address unit drains, and the MFMA pipe with
  // it.  Stage j + 1 must have landed by the barrier of stage j.
  constexpr int H1 = C::LPS / 2;  // loads of a stage issued in its first slot
  zero_acc();
  ld_setup(first);
  ld_kstep();
  for (int s = 0; s < C::NS; ++s) {
    const int n = s + 1 < C::NS ? C::LPS : H1;
    for (int l = 0; l < n; ++l) load_one(s, l);
    if (s + 1 < C::NS) ld_advance();
  }
  // in flight: stages 0 .. NS-2 whole and the first half of stage NS - 1
  __builtin_amdgcn_s_waitcnt(wait_vm((C::NS - 2) * C::LPS + H1));  // own stage-0 loads landed
  phase_barrier();
  read_frags(0, 0, 0);
  int j = 0;
  for (int t = first; t < total_tiles; t += gridDim.x) {
    for (int kb = 0; kb < nkb; ++kb, ++j) {
      const int buf = j & (C::NS - 1);
      const int pbuf = (j + C::NS - 1) & (C::NS - 1);  // stage j + NS - 1 (= buffer of j - 1)
      // K-step 0: the second half of stage j + NS - 1's loads among its MFMAs
      read_frags(buf, 1, 1);
#pragma unroll
      for (int l = H1; l < C::LPS; ++l) load_one(pbuf, l);
      mfma_set(0);
      __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
#pragma unroll
      for (int l = H1; l < C::LPS; ++l) {
        __builtin_amdgcn_sched_group_barrier(0x008, 16 / (C::LPS - H1), 0);
        __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
      ld_advance();  // to stage j + NS
#pragma unroll
      for (int ks = 1; ks < C::KSTEPS - 1; ++ks) {
        read_frags(buf, ks + 1, (ks + 1) & 1);
        mfma_set(ks & 1);
      }
      __builtin_amdgcn_sched_barrier(0);
      __builtin_amdgcn_s_waitcnt(wait_vm((C::NS - 2) * C::LPS));  // own stage j+1 landed
      __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
      phase_barrier();
      // last K-step: the first half of stage j + NS's loads among its MFMAs
      read_frags((j + 1) & (C::NS - 1), 0, 0);  // past the last stage: a harmless stale read
#pragma unroll
      for (int l = 0; l < H1; ++l) load_one(buf, l);
      mfma_set((C::KSTEPS - 1) & 1);
      __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
#pragma unroll
      for (int l = 0; l < H1; ++l) {
        __builtin_amdgcn_sched_group_barrier(0x008, 16 / H1, 0);
        __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    epilogue(tile_info(t));
    zero_acc();
  }
  __builtin_amdgcn_s_waitcnt(kWaitAll);
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
                                       hipFuncAttributeMaxDynamicSharedMemorySize, Stage::LDS);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  const long long m_tiles = (a.offsets ? static_cast<long long>(ceil_div(seg.total_rows, kBM)) + seg.groups
                                       : ceil_div(seg.static_rows, kBM));
  const long long tiles = m_tiles * ceil_div(a.N, OUT_COLS);
  if (tiles == 0) return hipSuccess;
  long long grid = std::min<long long>(tiles, device_cu_count());  // one workgroup per CU (LDS)
  grid = ((grid + 7) / 8) * 8;
  hipLaunchKernelGGL((tiled_kernel<GATED>), dim3(static_cast<unsigned>(grid)), dim3(kThreads), Stage::LDS, st, a);
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
