// Expert FFN for prefill-sized batches: a persistent bf16 MFMA grouped GEMM
// with direct-to-LDS loads, two waves per SIMD.
//
// Tiles.  An output tile is 256 token rows x 256 weight rows of one group
// (expert).  For the gate/up GEMM the 256 weight rows are 128 gate rows and
// the 128 up rows of the same output columns, so a tile yields 128 columns of
// h = silu(gate) * up.  Tiles are numbered group-major, then by n-tile, then
// by m-tile (a launch of static rows alone: in blocks of 8 m-tiles, see
// SBLK), so the m-tiles that share a weight tile are neighbours; each
// XCD (workgroups are dealt round-robin to the 8 XCDs) owns a contiguous run
// of tile ids, walked t, t + gridDim, ... by its workgroups, so they run side
// by side on one XCD and the weights cross the fabric once.  The group of a
// tile comes from the device-side offsets: every workgroup holds the groups'
// m-tile prefix in registers (lane L, entry i: group L + 64 i) and counts the
// groups that end at or before the tile.  Group sizes never leave the
// device.
//
// Tail tiles.  An expert whose rows past its last whole m-tile number 1..128
// takes them in tiles of 128 token rows, with their own LDS layout and
// pipeline (see TAIL): half the MFMA work per row of a padded 256-row
// m-tile.
//
// Two problems.  The shared experts (static rows: every token) can run in
// the routed experts' launch: their tiles come first, and each load stream
// and the epilogue follow the problem of the tile they are on.  This is used
// when the shared tiles alone would leave a partly filled last round.  The
// routed experts' tail tiles (gated projection) come after them; a
// workgroup's run of tiles then holds one problem only, so that within it
// neither the loads nor the epilogue select a problem per tile.
//
// Waves.  Eight waves, two per SIMD; wave (wm, wn) owns token rows
// 64*wm .. +63 and weight rows 128*wn .. +127 of the tile: 2 x 4
// v_mfma_f32_32x32x16_bf16 tiles (weights as the A operand, tokens as B),
// 128 fp32 accumulators.  Two waves per SIMD let one wave's MFMAs run while
// the other waits to issue a load: with one wave per SIMD (128 x 128 each,
// half the LDS reads per MFMA) the MFMA pipe idled during every such stall.
//
// Stages.  K advances in stages of 64.  A stage is an X part [256 x 64] and
// a W part [256 x 64] (128-byte rows, 32 KB each), filled by
// buffer_load_dwordx4 ... lds, which writes 64 lanes x 16 bytes to
// consecutive LDS addresses without passing through registers; a load
// covers 8 whole 128-byte rows, the access the vector L1 serves fastest.
// Part P (X of stage s: 2s, W of stage s: 2s + 1) lives in slot P mod 5 of
// a ring of five parts, all 160 KB of LDS.  Chunk c (16 bytes) of LDS row r
// sits at slot c ^ ((r >> 1) & 7): every lane of a load fetches the global
// chunk that belongs at its fixed LDS slot, and the 16 rows that 16 lanes of
// an MFMA fragment read land in 16 distinct bank groups.  Rows past a
// group's end, columns past N and the K tail get byte offsets >= 2^31, past
// the buffer descriptor's range: they read as zeros and cost no memory
// traffic.
//
// Pipeline.  One workgroup barrier per stage, placed before its last K-step
// after each wave has waited for its own loads of the next stage and for its
// LDS reads: past barrier j the slot of X of stage j takes W of stage j + 2
// (issued among the MFMAs of stage j's last K-step and stage j + 1's first)
// and the slot of W of stage j takes X of stage j + 3 (issued among the
// MFMAs of stage j + 1's K-steps 1 and 2): two loads per wave and K-step.  The
// stage sequence runs on across tile boundaries.
//
// Epilogue.  A lane holds row r, columns 8*v + 4*h + 0..3 (v < 4, h = lane
// half) of each 32 x 32 accumulator tile.  Values are converted in bf16
// pairs; the down projection stages them through 4 KB of LDS per wave (free
// during the epilogue) so that each 16-byte store instruction writes eight
// whole 128-byte lines, the gated projection stores them directly after a
// swap between the lane halves.
#include "ffn_impl.h"

namespace moe {
namespace {

constexpr int kBM = 256;             // token rows per tile
constexpr int kBN = 256;             // weight rows per tile
constexpr int kThreads = 8 * kWave;  // eight waves, two per SIMD
constexpr int kMaxGroups = 1024;
constexpr int kHalfTailK = 4096;  // K from which grouped launches take half tail tiles
constexpr int kBlockM = 8;           // m-tiles per block of a static group's tile order

// One K stage and the ring of its parts.
struct Stage {
  static constexpr int BK = 64;              // K per stage
  static constexpr int CPR = BK * 2 / 16;    // 16-byte chunks per LDS row
  static constexpr int RPI = kWave / CPR;    // rows per load instruction
  static constexpr int SWZ = 16 / CPR;       // rows sharing one swizzle key
  static constexpr int ROW = BK * 2;         // bytes per LDS row
  static constexpr int PART = kBM * ROW;     // one operand of a stage: 32 KB
  static constexpr int NPARTS = 5;           // ring slots
  static constexpr int LDS = NPARTS * PART;  // 160 KB, all of it
  static constexpr int LPP = 32 / RPI;       // loads per part per wave
  static constexpr int KSTEPS = BK / 16;     // MFMA K-steps per stage
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

__device__ __forceinline__ int wave_sum(int v) {
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) v += __shfl_xor(v, off);
  return v;
}
__device__ __forceinline__ int wave_max(int v) {
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) v = max(v, __shfl_xor(v, off));
  return v;
}
__device__ __forceinline__ int wave_min(int v) {
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) v = min(v, __shfl_xor(v, off));
  return v;
}

// An element of an index array that the kernel only reads, at a uniform
// index, through the constant address space: a scalar load.  Its wait
// (lgkmcnt) leaves the vector-memory counter alone; a vector load here would
// be waited for with that counter, which completes in order, and so drain
// every tile load and output store in flight.
typedef const int __attribute__((address_space(4)))* ConstIntPtr;
__device__ __forceinline__ int load_uniform(const int* p, int i) {
  return ((ConstIntPtr)(uintptr_t)p)[i];
}

template <bool B>
struct Half {
  static constexpr bool value = B;
};
// the problem of a run of full tiles: 0 (sp), 1 (g) or -1 (each tile its own)
template <int P>
struct Sel {
  static constexpr int value = P;
};

// Two GEMMs of one kind in one launch: the tiles of sp (static rows, e.g. the
// shared experts over every token; sp_tiles of them, 0 when absent) come
// first, then those of g (the routed experts).  One grid keeps every CU busy
// across both: neither leaves a partly filled last round on its own.
struct TiledArgs {
  GemmArgs g;
  GemmArgs sp;
  int sp_tiles;
};

// PAIR = false compiles the one-problem kernel: every problem selection
// below folds to g.  SBLK (one problem of static rows only, e.g. the shared
// experts in a launch of their own) orders its tiles in blocks of kBlockM
// m-tiles, n-tile-major inside a block: one XCD's 32 concurrent tiles are
// then 8 m-tiles x 4 n-tiles, instead of 32 m-tiles of one n-tile, each of
// whose token tiles would be fetched again for every n-tile.
//
// TAIL (grouped problems): a group whose rows past its last whole 256-row
// m-tile number 1..128 runs them as tail tiles of 128 token rows, half the
// MFMA work of a padded m-tile, in one of two shapes with their own LDS
// layouts and pipelines.  A workgroup drains its pipeline where its sequence
// of tiles switches between full and tail tiles.
//  - TAIL 1, wide: 128 x 512 weight rows (two column tiles).  Within a group
//    the tiles go by pairs of column tiles: the full tiles of column tiles 2p
//    and 2p + 1 (m-tiles fastest), then the tail tile that covers both.
//    Two 80 KB stages: X [128 x 64], W [512 x 64].
//  - TAIL 2, half: 128 x 256 weight rows.  Within a group the tiles go by
//    column tiles, m-tiles fastest, the tail tile last.  Three 48 KB stages:
//    X [128 x 64], W [256 x 64].  On long K a wide tail tile, with 80 KB
//    per stage, waits on weight rows that miss L2 and takes 1.28 times a
//    full tile; a half tile takes 0.58 times a full tile for half its work.
template <bool GATED, int kPfx, bool PAIR, bool SBLK, int TAIL>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2))) void tiled_kernel(TiledArgs ta) {
  using C = Stage;
  const GemmArgs& a = ta.g;
  const GemmArgs& sp = ta.sp;
  const int sp_tiles = PAIR ? ta.sp_tiles : 0;
  constexpr int OUT_COLS = GATED ? kBN / 2 : kBN;
  constexpr uint32_t kInvalid = 0x80000000u;
  constexpr int kRecords = 0x7fffffff;
  constexpr int kRsrcWord3 = 0x00020000;

  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];

  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int wm = wave & 3, wn = wave >> 2;
  const int lrow = lane & 31, lhalf = lane >> 5;
  const int n_tiles_n = ceil_div(a.N, OUT_COLS);
  const int n_tiles_t = ceil_div(n_tiles_n, 2);  // column tiles of a wide tail tile (512 weight rows)

  // full m-tiles and tail tiles of a group of n rows
  auto group_shape = [&](int n, int& fm, int& tl) {
    const int rem = n % kBM;
    tl = (TAIL && rem > 0 && rem <= kBM / 2) ? 1 : 0;
    fm = n / kBM + ((rem > 0 && !tl) ? 1 : 0);
  };
  // tile prefix of the groups, in registers: lane L holds the end (one past
  // the last tile; without TAIL, the last m-tile) of groups L + 64 i,
  // i < kPfx; groups past the end hold INT_MAX
  int mt_end[kPfx];
  int total_mt;
  if (a.offsets == nullptr) {
    total_mt = ceil_div(a.static_rows, kBM);
#pragma unroll
    for (int i = 0; i < kPfx; ++i) mt_end[i] = 0x7fffffff;
  } else {
    int carry = 0;
#pragma unroll
    for (int i = 0; i < kPfx; ++i) {
      const int g = i * kWave + lane;
      int cnt = 0;
      if (i * kWave < a.groups && g < a.groups) {
        const int n = a.offsets[g + 1] - a.offsets[g];
        if constexpr (TAIL) {
          int fm, tl;
          group_shape(n, fm, tl);
          cnt = TAIL == 1 ? fm * n_tiles_n + tl * n_tiles_t : (fm + tl) * n_tiles_n;
        } else {
          cnt = ceil_div(n, kBM);
        }
      }
      int inc = cnt;
#pragma unroll
      for (int off = 1; off < kWave; off <<= 1) {
        const int o = __shfl_up(inc, off);
        if (lane >= off) inc += o;
      }
      mt_end[i] = g < a.groups ? carry + inc : 0x7fffffff;
      carry += __shfl(inc, kWave - 1);
    }
    total_mt = __builtin_amdgcn_readfirstlane(carry);  // equal in every lane; the compiler cannot tell
  }
  // tiles of g: with TAIL the prefix already counts tiles
  const int total_tiles = sp_tiles + ((TAIL && a.offsets != nullptr) ? total_mt : total_mt * n_tiles_n);
  const int per_xcd = gridDim.x / 8;
  const int first = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
  if (first >= total_tiles) return;
  const int sp_mt = sp_tiles > 0 ? ceil_div(sp.static_rows, kBM) : 1;

  struct TileInfo {
    int p, g, row_base, m, m0, nt;  // p: 0 for sp, 1 for g
    bool tail;                      // a tail tile (wide tails: nt counts 512-row column tiles)
  };
  // group of tile t: the number of groups whose tiles all precede t
  auto tile_info = [&](int t_all) {
    // tile ids are wave-uniform: stated here, every branch on them is uniform
    // and so are the buffer descriptors built from the tile (else the
    // compiler wraps each load in a loop over the lanes' descriptors)
    t_all = __builtin_amdgcn_readfirstlane(t_all);
    TileInfo ti;
    ti.tail = false;
    ti.p = (PAIR && t_all < sp_tiles) ? 0 : 1;
    const int t = ti.p ? t_all - sp_tiles : t_all;
    int mg = ti.p ? total_mt : sp_mt, base = 0;
    ti.g = 0;
    ti.row_base = 0;
    ti.m = ti.p ? a.static_rows : sp.static_rows;
    if (ti.p && a.offsets != nullptr) {
      constexpr int kScale = 1;
      const int scale = TAIL ? kScale : n_tiles_n;
      int cnt = 0, lo = 0, hi = 0x7fffffff;
#pragma unroll
      for (int i = 0; i < kPfx; ++i) {
        const int e = mt_end[i];
        const bool before = e != 0x7fffffff && e * scale <= t;
        cnt += before ? 1 : 0;
        lo = before ? max(lo, e) : lo;
        hi = before ? hi : min(hi, e);
      }
      cnt = wave_sum(cnt);
      lo = wave_max(lo);
      hi = wave_min(hi);
      const int g = __builtin_amdgcn_readfirstlane(cnt);
      ti.g = g;
      ti.row_base = load_uniform(a.offsets, g);
      ti.m = load_uniform(a.offsets, g + 1) - ti.row_base;
      base = __builtin_amdgcn_readfirstlane(lo) * scale;
      mg = __builtin_amdgcn_readfirstlane(hi) - __builtin_amdgcn_readfirstlane(lo);
      if constexpr (TAIL) {
        int fm, tl;
        group_shape(ti.m, fm, tl);
        const int local = t - base;
        if constexpr (TAIL == 1) {
          // pairs of column tiles: the full tiles of columns 2p and 2p + 1
          // (m-tiles fastest), then the tail tile of pair p
          const int per_pair = 2 * fm + tl;
          const int pr = min(local / max(per_pair, 1), n_tiles_t - 1);
          const int r = local - pr * per_pair;
          const int nfull = min(2, n_tiles_n - 2 * pr) * fm;
          const int fmd = max(fm, 1);
          ti.tail = r >= nfull;
          ti.nt = ti.tail ? pr : 2 * pr + r / fmd;
          ti.m0 = (ti.tail ? fm : r % fmd) * kBM;
        } else {
          // column tiles in order; within one, the full m-tiles, then the
          // tail tile of the same weight rows
          const int per_col = fm + tl;
          const int c = local / max(per_col, 1);
          const int r = local - c * per_col;
          ti.tail = tl && r == fm;
          ti.nt = c;
          ti.m0 = r * kBM;
        }
        ti.tail = __builtin_amdgcn_readfirstlane(ti.tail ? 1 : 0) != 0;
        ti.p = 1;
        ti.g = __builtin_amdgcn_readfirstlane(ti.g);
        ti.row_base = __builtin_amdgcn_readfirstlane(ti.row_base);
        ti.m = __builtin_amdgcn_readfirstlane(ti.m);
        ti.m0 = __builtin_amdgcn_readfirstlane(ti.m0);
        ti.nt = __builtin_amdgcn_readfirstlane(ti.nt);
        return ti;
      }
    }
    const int local = t - base;
    if constexpr (SBLK) {
      const int mfull = (mg / kBlockM) * kBlockM;
      const int full_tiles = mfull * n_tiles_n;
      if (local < full_tiles) {
        const int b = local / (kBlockM * n_tiles_n);
        const int r = local - b * (kBlockM * n_tiles_n);
        ti.nt = r / kBlockM;
        ti.m0 = (b * kBlockM + (r - ti.nt * kBlockM)) * kBM;
      } else {
        const int mr = mg - mfull;
        const int r = local - full_tiles;
        ti.nt = r / mr;
        ti.m0 = (mfull + (r - ti.nt * mr)) * kBM;
      }
    } else {
      ti.nt = local / mg;
      ti.m0 = (local - ti.nt * mg) * kBM;
    }
    if (PAIR) ti.p = __builtin_amdgcn_readfirstlane(ti.p);
    ti.g = __builtin_amdgcn_readfirstlane(ti.g);
    ti.row_base = __builtin_amdgcn_readfirstlane(ti.row_base);
    ti.m = __builtin_amdgcn_readfirstlane(ti.m);
    ti.m0 = __builtin_amdgcn_readfirstlane(ti.m0);
    ti.nt = __builtin_amdgcn_readfirstlane(ti.nt);
    return ti;
  };

  // ---- load side ----
  // Two streams, X one stage ahead of W.  Wave w fills rows 32w..32w+31 of
  // a part; load i writes rows 32w + 8i + lane/8, slot lane%8, fetching
  // the global chunk slot ^ ((row / 2) % 8).
  auto chunk_of = [&](int i, int ln) {
    const int r = 32 * wave + C::RPI * i + ln / C::CPR;
    return (ln % C::CPR) ^ ((r / C::SWZ) % C::CPR);
  };
  // the 32 weight rows of this wave are all gate rows or all up rows
  const bool w_up = GATED && ((wave >> 1) & 1);
  // the workgroup's current run of tiles of one kind: its first tile and the
  // first tile of its sequence past the run (loads past it are dead: no
  // traffic)
  int run_start = first, run_end = total_tiles;
  // (through ta: a selection between two captured references would index the
  // closure at run time and keep the kernel's arguments in scratch memory)
  auto prob = [&](int p) -> const GemmArgs& { return (!PAIR || p) ? ta.g : ta.sp; };
  const int nkb_g = ceil_div(a.K, C::BK);
  auto kmask = [&](int kb, int p, int K) { return kb * C::BK + chunk_of(p, lane) * 8 < K ? 0u : kInvalid; };
  // part P (X of stage s: 2s, W of stage s: 2s + 1) lives in slot P % 5
  auto part_ptr = [&](int P) { return smem + (P % C::NPARTS) * C::PART; };
  // ---- compute side ----
  const int xrow0 = wm * 64, wrow0 = wn * 128;
  const int rsw = (lrow / C::SWZ) % C::CPR;
  bf16x8 xf[2][2], wf[2][4];
  f32x16 acc[4][2];
  auto read_frags = [&](int s, int ks, int set) {
    const unsigned char* xp = part_ptr(2 * s);
    const unsigned char* wp = part_ptr(2 * s + 1);
    const int slot = ((2 * ks + lhalf) ^ rsw) << 4;
#pragma unroll
    for (int t = 0; t < 4; ++t)
      wf[set][t] = as_bf16x8(*reinterpret_cast<const u32x4*>(wp + (wrow0 + t * 32 + lrow) * C::ROW + slot));
#pragma unroll
    for (int t = 0; t < 2; ++t)
      xf[set][t] = as_bf16x8(*reinterpret_cast<const u32x4*>(xp + (xrow0 + t * 32 + lrow) * C::ROW + slot));
  };
  auto mfma_set = [&](int set) {
#pragma unroll
    for (int tn = 0; tn < 4; ++tn)
#pragma unroll
      for (int tm = 0; tm < 2; ++tm) acc[tn][tm] = mfma32x32x16(wf[set][tn], xf[set][tm], acc[tn][tm]);
  };
  auto zero_acc = [&]() {
#pragma unroll
    for (int tn = 0; tn < 4; ++tn)
#pragma unroll
      for (int tm = 0; tm < 2; ++tm) acc[tn][tm] = f32x16{};
  };
  // the wave's output columns: WCOLS of them from col_w; rows from xr0
  constexpr int WCOLS = GATED ? 64 : 128;
  // Epilogue.  The down projection's wave writes 128 columns per row: its
  // outputs go through scr, 4 KB of LDS that only this wave touches until it
  // issues its next loads, so that every store instruction writes eight
  // whole 128-byte lines.  Per row group (32 rows) and pair of 32-column
  // tiles the lanes write their converted values (row erow, columns
  // 8 v4 + 4 ehalf .. +3 of each tile) into a block of 32 rows of 128 bytes,
  // 16-byte chunk c of row r at slot c ^ (r & 7), then read it back by rows
  // (lane L: chunk L % 8 of row 8 q + L / 8) and store.  The gated
  // projection's wave writes half as many columns from twice the
  // accumulators; there a swap between the lane halves gives each lane 8
  // consecutive columns and the stores go straight out (measured faster than
  // staging for it).
  // A half tile's wave (tail tiles, Half<true>) holds 2 x 2 accumulator
  // tiles: 32 output columns (gated: gate in tile 0, up in tile 1) or 64.
  auto epilogue = [&](auto half, const TileInfo& ti, const GemmArgs& pr, int xr0, int col_w, unsigned char* scr) {
    constexpr bool kHalf = decltype(half)::value;
    constexpr int kUp = kHalf ? 1 : 2;       // accumulator tile of the up rows of tile tn: tn + kUp
    constexpr int kGroups = kHalf ? 1 : 2;   // 32-column tiles (gated) or 64-column pairs (down) per wave
    const int ln = opaque_lane_id();
    const int erow = ln & 31, ehalf = ln >> 5;
    // The tile's output rows through a buffer descriptor: rows past the
    // group and columns past N get offsets >= 2^31, which the hardware
    // drops, so the stores need no branches.
    const __amdgpu_buffer_rsrc_t rs_o = __builtin_amdgcn_make_buffer_rsrc(
        pr.out + static_cast<size_t>(ti.row_base + ti.m0) * pr.N, 0, kRecords, kRsrcWord3);
    // pk[2 v4 + h]: columns 8 v4 + 4 ehalf + 2 h, +1 of accumulator tile (tn, tm)
    auto convert = [&](int tn, int tm, uint32_t (&pk)[8]) {
#pragma unroll
      for (int v4 = 0; v4 < 4; ++v4) {
        float o[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float c0 = acc[tn][tm][4 * v4 + i];
          if constexpr (GATED)
            o[i] = silu(c0) * acc[tn + kUp][tm][4 * v4 + i];
          else
            o[i] = c0;
        }
        pk[2 * v4] = cvt_pk_bf16(o[0], o[1]);
        pk[2 * v4 + 1] = cvt_pk_bf16(o[2], o[3]);
      }
    };
#pragma unroll
    for (int tm = 0; tm < 2; ++tm) {
      if constexpr (GATED) {
        const int r = xr0 + tm * 32 + erow;  // row within the tile
        const uint32_t row_off = ti.m0 + r < ti.m ? static_cast<uint32_t>(r * pr.N * 2) : kInvalid;
#pragma unroll
        for (int tn = 0; tn < kGroups; ++tn) {
          uint32_t pk[8];
          convert(tn, tm, pk);
#pragma unroll
          for (int q = 0; q < 2; ++q) {  // columns 16q .. 16q+15 of the 32-column tile
            // lower lanes keep columns 16q+0..3 and take 16q+4..7 from the
            // upper half; upper lanes take 16q+8..11 and keep 16q+12..15
            const auto s0 = __builtin_amdgcn_permlane32_swap(pk[4 * q], pk[4 * q + 2], false, false);
            const auto s1 = __builtin_amdgcn_permlane32_swap(pk[4 * q + 1], pk[4 * q + 3], false, false);
            const u32x4 v = {s0[0], s1[0], s0[1], s1[1]};
            const int col = col_w + tn * 32 + 16 * q + 8 * ehalf;
            const uint32_t off = col < pr.N ? row_off + static_cast<uint32_t>(col * 2) : kInvalid;
            __builtin_amdgcn_raw_buffer_store_b128(v, rs_o, off | (row_off & kInvalid), 0, 0);
          }
        }
      } else {
#pragma unroll
        for (int tp = 0; tp < kGroups; ++tp) {
#pragma unroll
          for (int a2 = 0; a2 < 2; ++a2) {
            uint32_t pk[8];
            convert(2 * tp + a2, tm, pk);
#pragma unroll
            for (int v4 = 0; v4 < 4; ++v4) {
              const int chunk = 4 * a2 + v4;  // columns 32 a2 + 8 v4 .. of the pair
              typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
              *reinterpret_cast<u32x2*>(scr + erow * 128 + ((chunk ^ (erow & 7)) << 4) + 8 * ehalf) =
                  u32x2{pk[2 * v4], pk[2 * v4 + 1]};
            }
          }
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int rr = 8 * q + (ln >> 3), c = ln & 7;
            const u32x4 v = *reinterpret_cast<const u32x4*>(scr + rr * 128 + ((c ^ (rr & 7)) << 4));
            const int r = xr0 + tm * 32 + rr;  // row within the tile
            const int col = col_w + tp * 64 + 8 * c;
            const uint32_t off =
                (ti.m0 + r < ti.m && col < pr.N) ? static_cast<uint32_t>(r * pr.N * 2 + col * 2) : kInvalid;
            __builtin_amdgcn_raw_buffer_store_b128(v, rs_o, off, 0, 0);
          }
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // ---- pipeline of full tiles ----
  // Stage j: barrier before its last K-step, after every wave's last LDS
  // read of the stage.  Past barrier j - 1 the slot of X of stage j - 1
  // takes W of stage j + 1 (first half among the MFMAs of stage j - 1's last
  // K-step, second half among those of stage j's first) and the slot of W
  // of stage j - 1 takes X of stage j + 2 (among the MFMAs of stage j's
  // K-steps 1 and 2).  Before barrier j each wave waits for its loads of
  // stage j + 1; only X of stage j + 2 may still be in flight.
  auto full_run = [&](auto prob_sel) {
    // kP: the problem of every tile of the run (0: sp, 1: g), or -1 when the
    // run takes both and each tile selects its own
    constexpr int kP = decltype(prob_sel)::value;
    auto pick = [&](int p) { return kP >= 0 ? kP : (PAIR ? p : 1); };
    __amdgpu_buffer_rsrc_t rs_x, rs_w;
    uint32_t xoff[C::LPP], woff[C::LPP];
    int x_tile = first, x_kb = 0, w_tile = first, w_kb = 0;
    int x_p = 1, w_p = 1, x_nkb = 1, w_nkb = 1;  // each stream's problem and its K stages
    uint32_t kx0 = 0, kx1 = 0, kw0 = 0, kw1 = 0;

    // The gathered source rows (x_rows) of the X stream's next tile are
    // loaded one tile ahead, so that waiting for them never waits for the
    // tile loads in flight (the vector-memory counter completes in order).
    int xr_next[C::LPP];
    auto x_rows_of = [&](int t, int (&xr)[C::LPP]) {
      const TileInfo ti = tile_info(t);
      const GemmArgs& q = prob(pick(ti.p));
      const int ln = opaque_lane_id();
      if (q.x_rows) {
#pragma unroll
        for (int i = 0; i < C::LPP; ++i) {
          const int r = 32 * wave + C::RPI * i + ln / C::CPR;
          xr[i] = q.x_rows[ti.row_base + (ti.m0 + r < ti.m ? ti.m0 + r : 0)];
        }
      }
    };
    // prefetched: xr_next holds the rows of t_in (loaded by the previous call)
    auto x_setup = [&](int t_in, bool prefetched) {
      const bool live = t_in < run_end;
      const int t = live ? t_in : run_start;
      const TileInfo ti = tile_info(t);
      x_p = pick(ti.p);
      const GemmArgs& q = prob(x_p);
      x_nkb = PAIR ? ceil_div(q.K, C::BK) : nkb_g;
      const int ln = opaque_lane_id();
      const uint16_t* xb = q.x_rows ? q.x : q.x + static_cast<size_t>(ti.row_base + ti.m0) * q.K;
      rs_x = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(xb), 0, kRecords, kRsrcWord3);
      int xr[C::LPP];
#pragma unroll
      for (int i = 0; i < C::LPP; ++i) xr[i] = 32 * wave + C::RPI * i + ln / C::CPR;
      if (q.x_rows) {
        if (live && !prefetched) x_rows_of(t, xr_next);
#pragma unroll
        for (int i = 0; i < C::LPP; ++i) xr[i] = xr_next[i];
      }
      // past the run (dead) the loads carry invalid offsets: no traffic
#pragma unroll
      for (int i = 0; i < C::LPP; ++i) {
        const int r = 32 * wave + C::RPI * i + ln / C::CPR;
        xoff[i] = (live && ti.m0 + r < ti.m) ? static_cast<uint32_t>(xr[i] * q.K * 2 + chunk_of(i, ln) * 16) : kInvalid;
      }
      if (t_in + static_cast<int>(gridDim.x) < run_end) x_rows_of(t_in + gridDim.x, xr_next);
    };
    auto w_setup = [&](int t_in) {
      const bool live = t_in < run_end;
      const uint32_t dead = live ? 0u : kInvalid;
      const int t = live ? t_in : run_start;
      const TileInfo ti = tile_info(t);
      w_p = pick(ti.p);
      const GemmArgs& q = prob(w_p);
      w_nkb = PAIR ? ceil_div(q.K, C::BK) : nkb_g;
      const int ln = opaque_lane_id();
      const int col0 = ti.nt * OUT_COLS;
      const size_t gofs = static_cast<size_t>(ti.g) * q.group_stride + static_cast<size_t>(col0) * q.ldw;
      rs_w = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>((w_up ? q.w1 : q.w0) + gofs), 0, kRecords, kRsrcWord3);
#pragma unroll
      for (int i = 0; i < C::LPP; ++i) {
        const int r = 32 * wave + C::RPI * i + ln / C::CPR;
        const int lcol = GATED ? (r >> 7) * 64 + (r & 63) : r;
        woff[i] = ((col0 + lcol < q.N) ? static_cast<uint32_t>(lcol * q.ldw * 2 + chunk_of(i, ln) * 16) : kInvalid) | dead;
      }
    };
    auto x_kstep = [&]() {
      const uint32_t k = static_cast<uint32_t>(x_kb * C::BK * 2);
      const int K = prob(x_p).K;
      kx0 = k | kmask(x_kb, 0, K);
      kx1 = k | kmask(x_kb, 1, K);
    };
    auto w_kone = [&](int p) -> uint32_t {
      const GemmArgs& q = prob(w_p);
      const int k0 = w_kb * C::BK;
      uint32_t w;
      if (q.kseg >= q.K) {
        w = static_cast<uint32_t>(k0 * 2);
      } else if (q.kseg % C::BK == 0) {
        const int seg = k0 / q.kseg;
        w = static_cast<uint32_t>((static_cast<size_t>(seg) * q.seg_stride + (k0 - seg * q.kseg)) * 2);
      } else {
        const int kk = min(k0 + chunk_of(p, lane) * 8, q.K - 8);
        w = static_cast<uint32_t>((weight_col_offset(q, kk) - static_cast<size_t>(kk - k0)) * 2);
      }
      return w | kmask(w_kb, p, q.K);
    };
    auto w_kstep = [&]() {
      kw0 = w_kone(0);
      kw1 = w_kone(1);
    };
    auto x_advance = [&]() {
      if (++x_kb == (PAIR ? x_nkb : nkb_g)) {
        x_kb = 0;
        x_tile += gridDim.x;
        x_setup(x_tile, true);
      }
      x_kstep();
    };
    auto w_advance = [&]() {
      if (++w_kb == (PAIR ? w_nkb : nkb_g)) {
        w_kb = 0;
        w_tile += gridDim.x;
        w_setup(w_tile);
      }
      w_kstep();
    };
    auto x_load = [&](int s, int i) {
      const uint32_t k = (i & 1) ? kx1 : kx0;
      load_lds16(rs_x, part_ptr(2 * s) + wave * (32 * C::ROW) + i * 1024, (xoff[i] + k) | (k & kInvalid));
    };
    auto w_load = [&](int s, int i) {
      const uint32_t k = (i & 1) ? kw1 : kw0;
      load_lds16(rs_w, part_ptr(2 * s + 1) + wave * (32 * C::ROW) + i * 1024, (woff[i] + k) | (k & kInvalid));
    };
    zero_acc();
    x_tile = w_tile = run_start;
    x_kb = w_kb = 0;
    x_setup(run_start, false);
    x_kstep();
    w_setup(run_start);
    w_kstep();
    // stages 0 and 1, but only the first half of W of stage 1 (its second
    // half goes out with stage 0's first K-step)
    for (int s = 0; s < 2; ++s) {
#pragma unroll
      for (int i = 0; i < C::LPP; ++i) x_load(s, i);
      x_advance();
#pragma unroll
      for (int i = 0; i < C::LPP; ++i)
        if (s == 0 || i < C::LPP / 2) w_load(s, i);
      if (s == 0) w_advance();
    }
    __builtin_amdgcn_s_waitcnt(wait_vm(C::LPP + C::LPP / 2));  // own stage-0 loads landed
    phase_barrier();
    read_frags(0, 0, 0);
    int j = 0;
    for (int t = run_start; t < run_end; t += gridDim.x) {
      const TileInfo cur = tile_info(t);  // scalars, held through the K loop
      const int nkb = PAIR ? ceil_div(prob(pick(cur.p)).K, C::BK) : nkb_g;
      for (int kb = 0; kb < nkb; ++kb, ++j) {
        // K-step 0 with the second half of W of stage j + 1, K-steps 1 and 2
        // with X of stage j + 2: two loads per wave and K-step
#pragma unroll
        for (int ks = 0; ks < C::KSTEPS - 1; ++ks) {
          read_frags(j, ks + 1, (ks + 1) & 1);
#pragma unroll
          for (int i = 0; i < C::LPP / 2; ++i) {
            if (ks == 0)
              w_load(j + 1, C::LPP / 2 + i);
            else
              x_load(j + 2, (ks - 1) * (C::LPP / 2) + i);
          }
          if (ks == 0) w_advance();
          mfma_set(ks & 1);
          __builtin_amdgcn_sched_barrier(0);
        }
        x_advance();
        __builtin_amdgcn_s_waitcnt(wait_vm(C::LPP));  // own stage j+1 landed
        __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
        phase_barrier();
        // last K-step with the first half of W of stage j + 2
        read_frags(j + 1, 0, 0);  // past the last stage: a harmless stale read
#pragma unroll
        for (int i = 0; i < C::LPP / 2; ++i) w_load(j + 2, i);
        mfma_set((C::KSTEPS - 1) & 1);
        __builtin_amdgcn_sched_barrier(0);
      }
      // the W part of the tile's last stage is free until this wave loads X
      // of the stage three ahead into its own 4 KB of it
      epilogue(Half<false>{}, cur, prob(pick(cur.p)), xrow0, cur.nt * OUT_COLS + wn * WCOLS, part_ptr(2 * (j - 1) + 1) + wave * 4096);
      zero_acc();
    }
  };

  // ---- wide tail tiles (TAIL 1): 128 token rows x 512 weight rows ----
  // Two stages of 80 KB: X [128 rows x 128 B] at 0, W [512 rows x 128 B] at
  // 16 KB, the same chunk swizzle as the full parts.  Wave w fills X rows
  // 16w .. 16w+15 (two loads) and W rows 64w .. 64w+63 (eight loads, all
  // gate or all up rows); wave (wm_t, wn_t) = (w & 1, w >> 1) owns token rows
  // 64 wm_t .. +63 and weight rows 128 wn_t .. +127, the same 2 x 4 MFMA
  // tiles as in a full tile.  The loads of stage j + 1 go out among the
  // first MFMAs of stage j into the other stage buffer, read last in stage
  // j - 1.  (Stages of 32 along K, four in flight in 40 KB buffers, were
  // measured no faster.)
  auto tail_run_wide = [&]() {
    constexpr int T_XROWS = kBM / 2, T_WROWS = 2 * kBN;
    constexpr int T_XPART = T_XROWS * C::ROW;             // 16 KB
    constexpr int T_STAGE = T_XPART + T_WROWS * C::ROW;   // 80 KB
    constexpr int T_XL = T_XROWS / C::RPI / 8;            // X loads per wave and stage: 2
    constexpr int T_WL = T_WROWS / C::RPI / 8;            // W loads per wave and stage: 8
    constexpr int OUT_COLS_T = 2 * OUT_COLS;
    static_assert(2 * T_STAGE <= C::LDS, "two tail stages fit the LDS");
    const int wm_t = wave & 1, wn_t = wave >> 1;
    const int xrow0_t = wm_t * 64, wrow0_t = wn_t * 128;
    auto t_buf = [&](int b) { return smem + b * T_STAGE; };
    auto t_read_frags = [&](int b, int ks, int set) {
      const unsigned char* xp = t_buf(b);
      const unsigned char* wp = xp + T_XPART;
      const int slot = ((2 * ks + lhalf) ^ rsw) << 4;
  #pragma unroll
      for (int t = 0; t < 4; ++t)
        wf[set][t] = as_bf16x8(*reinterpret_cast<const u32x4*>(wp + (wrow0_t + t * 32 + lrow) * C::ROW + slot));
  #pragma unroll
      for (int t = 0; t < 2; ++t)
        xf[set][t] = as_bf16x8(*reinterpret_cast<const u32x4*>(xp + (xrow0_t + t * 32 + lrow) * C::ROW + slot));
    };
    auto run = [&]() {
      __amdgpu_buffer_rsrc_t trs_x, trs_w;
      uint32_t txoff[T_XL], twoff[T_WL];
      int tt = first, tkb = 0;
      uint32_t tk0 = 0, tk1 = 0;
      // gathered source rows one tile ahead, as for the full tiles
      int txr_next[T_XL];
      auto t_rows_of = [&](int t) {
        const TileInfo ti = tile_info(t);
        const int ln = opaque_lane_id();
  #pragma unroll
        for (int i = 0; i < T_XL; ++i) {
          const int r = 16 * wave + C::RPI * i + ln / C::CPR;
          txr_next[i] = a.x_rows[ti.row_base + (ti.m0 + r < ti.m ? ti.m0 + r : 0)];
        }
      };
      auto t_setup = [&](int t_in, bool prefetched) {
        const bool live = t_in < run_end;
        const uint32_t dead = live ? 0u : kInvalid;
        const TileInfo ti = tile_info(live ? t_in : run_start);
        const int ln = opaque_lane_id();
        const uint16_t* xb = a.x_rows ? a.x : a.x + static_cast<size_t>(ti.row_base + ti.m0) * a.K;
        trs_x = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(xb), 0, kRecords, kRsrcWord3);
        if (a.x_rows && live && !prefetched) t_rows_of(t_in);
  #pragma unroll
        for (int i = 0; i < T_XL; ++i) {
          const int r = 16 * wave + C::RPI * i + ln / C::CPR;
          const int xr = a.x_rows ? txr_next[i] : r;
          txoff[i] = (live && ti.m0 + r < ti.m) ? static_cast<uint32_t>(xr * a.K * 2 + chunk_of(i, ln) * 16) : kInvalid;
        }
        if (a.x_rows && t_in + static_cast<int>(gridDim.x) < run_end) t_rows_of(t_in + gridDim.x);
        const int col0 = ti.nt * OUT_COLS_T;
        const size_t gofs = static_cast<size_t>(ti.g) * a.group_stride + static_cast<size_t>(col0) * a.ldw;
        const bool up = GATED && (wave & 1);  // W rows 64w .. 64w+63: gate rows for even w, up rows for odd w
        trs_w = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>((up ? a.w1 : a.w0) + gofs), 0, kRecords,
                                                  kRsrcWord3);
  #pragma unroll
        for (int i = 0; i < T_WL; ++i) {
          const int r = 64 * wave + C::RPI * i + ln / C::CPR;
          const int lcol = GATED ? (r >> 7) * 64 + (r & 63) : r;
          twoff[i] =
              ((col0 + lcol < a.N) ? static_cast<uint32_t>(lcol * a.ldw * 2 + chunk_of(i, ln) * 16) : kInvalid) | dead;
        }
      };
      auto t_kstep = [&]() {
        const uint32_t k = static_cast<uint32_t>(tkb * C::BK * 2);
        tk0 = k | kmask(tkb, 0, a.K);
        tk1 = k | kmask(tkb, 1, a.K);
      };
      auto t_advance = [&]() {
        if (++tkb == nkb_g) {
          tkb = 0;
          tt += gridDim.x;
          t_setup(tt, true);
        }
        t_kstep();
      };
      auto t_load = [&](int b, int i) {  // load i < T_XL: X, else W load i - T_XL
        const uint32_t k = (i & 1) ? tk1 : tk0;
        if (i < T_XL)
          load_lds16(trs_x, t_buf(b) + wave * (16 * C::ROW) + i * 1024, (txoff[i] + k) | (k & kInvalid));
        else
          load_lds16(trs_w, t_buf(b) + T_XPART + wave * (64 * C::ROW) + (i - T_XL) * 1024,
                     (twoff[i - T_XL] + k) | (k & kInvalid));
      };
      zero_acc();
      tt = run_start;
      tkb = 0;
      t_setup(tt, false);
      t_kstep();
  #pragma unroll
      for (int i = 0; i < T_XL + T_WL; ++i) t_load(0, i);
      t_advance();
      __builtin_amdgcn_s_waitcnt(kWaitAll);
      phase_barrier();
      int j = 0;
      for (int t = run_start; t < run_end; t += gridDim.x) {
        const TileInfo cur = tile_info(t);
        for (int kb = 0; kb < nkb_g; ++kb, ++j) {
          const int b = j & 1;
          t_read_frags(b, 0, 0);
  #pragma unroll
          for (int ks = 0; ks < C::KSTEPS; ++ks) {
            if (ks + 1 < C::KSTEPS) t_read_frags(b, ks + 1, (ks + 1) & 1);
            // stage j + 1's ten loads in the first three K-steps (4, 4, 2),
            // so that they have landed by the end of the stage
            constexpr int kFirst[5] = {0, 4, 8, 10, 10};
  #pragma unroll
            for (int i = kFirst[ks]; i < kFirst[ks + 1]; ++i) t_load(b ^ 1, i);
            mfma_set(ks & 1);
            __builtin_amdgcn_sched_barrier(0);
          }
          t_advance();
          __builtin_amdgcn_s_waitcnt(kWaitAll);  // own stage j+1 landed, LDS reads done
          phase_barrier();
        }
        // the buffer of the tile's last stage is free until the next loads
        // into it; this wave's own W rows there are its 8 KB
        epilogue(Half<false>{}, cur, a, xrow0_t, cur.nt * OUT_COLS_T + wn_t * WCOLS,
                 t_buf((j - 1) & 1) + T_XPART + wave * (64 * C::ROW));
        zero_acc();
      }
    };
    run();
  };

  // ---- half tail tiles (TAIL 2): 128 token rows x 256 weight rows ----
  // Stages of 48 KB, three in a ring: X [128 rows x 128 B] at 0, W [256
  // rows x 128 B] at 16 KB, the same chunk swizzle as the full parts.  Wave w
  // fills X rows 16w .. 16w+15 (two loads) and W rows 32w .. 32w+31 (four
  // loads, all gate or all up rows).  Gated, W row r holds the gate (r / 32
  // even) or up row of column 32 (r / 64) + r % 32, so that each 64-row
  // quarter holds the gate and up rows of 32 columns.  Wave (wm_t, wn_t) =
  // (w & 1, w >> 1) owns token rows 64 wm_t .. +63 and W rows 64 wn_t .. +63:
  // 2 x 2 MFMA tiles, half a full tile's work.  The loads of stage j + 2 go
  // out among the MFMAs of stage j into the buffer read last in stage j - 1;
  // before the barrier that ends stage j each wave waits for its loads of
  // stage j + 1.  A tail tile follows the full m-tiles of its column tile,
  // so it reads the same weight rows at about the same time.
  auto tail_run_half = [&]() {
    constexpr int T_XROWS = kBM / 2, T_WROWS = kBN;
    constexpr int T_XPART = T_XROWS * C::ROW;             // 16 KB
    constexpr int T_STAGE = T_XPART + T_WROWS * C::ROW;   // 48 KB
    constexpr int T_NBUF = 3;
    constexpr int T_XL = T_XROWS / C::RPI / 8;            // X loads per wave and stage: 2
    constexpr int T_WL = T_WROWS / C::RPI / 8;            // W loads per wave and stage: 4
    constexpr int T_LOADS = T_XL + T_WL;
    static_assert(T_NBUF * T_STAGE <= C::LDS, "three tail stages fit the LDS");
    const int wm_t = wave & 1, wn_t = wave >> 1;
    const int xrow0_t = wm_t * 64, wrow0_t = wn_t * 64;
    auto t_buf = [&](int s) { return smem + (s % T_NBUF) * T_STAGE; };
    auto t_read_frags = [&](int s, int ks, int set) {
      const unsigned char* xp = t_buf(s);
      const unsigned char* wp = xp + T_XPART;
      const int slot = ((2 * ks + lhalf) ^ rsw) << 4;
  #pragma unroll
      for (int t = 0; t < 2; ++t)
        wf[set][t] = as_bf16x8(*reinterpret_cast<const u32x4*>(wp + (wrow0_t + t * 32 + lrow) * C::ROW + slot));
  #pragma unroll
      for (int t = 0; t < 2; ++t)
        xf[set][t] = as_bf16x8(*reinterpret_cast<const u32x4*>(xp + (xrow0_t + t * 32 + lrow) * C::ROW + slot));
    };
    auto t_mfma_set = [&](int set) {
  #pragma unroll
      for (int tn = 0; tn < 2; ++tn)
  #pragma unroll
        for (int tm = 0; tm < 2; ++tm) acc[tn][tm] = mfma32x32x16(wf[set][tn], xf[set][tm], acc[tn][tm]);
    };
    auto run = [&]() {
      __amdgpu_buffer_rsrc_t trs_x, trs_w;
      uint32_t txoff[T_XL], twoff[T_WL];
      int tt = first, tkb = 0;
      uint32_t tk0 = 0, tk1 = 0;
      // gathered source rows one tile ahead, as for the full tiles
      int txr_next[T_XL];
      auto t_rows_of = [&](int t) {
        const TileInfo ti = tile_info(t);
        const int ln = opaque_lane_id();
  #pragma unroll
        for (int i = 0; i < T_XL; ++i) {
          const int r = 16 * wave + C::RPI * i + ln / C::CPR;
          txr_next[i] = a.x_rows[ti.row_base + (ti.m0 + r < ti.m ? ti.m0 + r : 0)];
        }
      };
      auto t_setup = [&](int t_in, bool prefetched) {
        const bool live = t_in < run_end;
        const uint32_t dead = live ? 0u : kInvalid;
        const TileInfo ti = tile_info(live ? t_in : run_start);
        const int ln = opaque_lane_id();
        const uint16_t* xb = a.x_rows ? a.x : a.x + static_cast<size_t>(ti.row_base + ti.m0) * a.K;
        trs_x = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(xb), 0, kRecords, kRsrcWord3);
        if (a.x_rows && live && !prefetched) t_rows_of(t_in);
  #pragma unroll
        for (int i = 0; i < T_XL; ++i) {
          const int r = 16 * wave + C::RPI * i + ln / C::CPR;
          const int xr = a.x_rows ? txr_next[i] : r;
          txoff[i] = (live && ti.m0 + r < ti.m) ? static_cast<uint32_t>(xr * a.K * 2 + chunk_of(i, ln) * 16) : kInvalid;
        }
        if (a.x_rows && t_in + static_cast<int>(gridDim.x) < run_end) t_rows_of(t_in + gridDim.x);
        const int col0 = ti.nt * OUT_COLS;
        const size_t gofs = static_cast<size_t>(ti.g) * a.group_stride + static_cast<size_t>(col0) * a.ldw;
        const bool up = GATED && (wave & 1);  // W rows 32w .. 32w+31: gate rows for even w, up rows for odd w
        trs_w = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>((up ? a.w1 : a.w0) + gofs), 0, kRecords,
                                                  kRsrcWord3);
  #pragma unroll
        for (int i = 0; i < T_WL; ++i) {
          const int r = 32 * wave + C::RPI * i + ln / C::CPR;
          const int lcol = GATED ? (r >> 6) * 32 + (r & 31) : r;
          twoff[i] =
              ((col0 + lcol < a.N) ? static_cast<uint32_t>(lcol * a.ldw * 2 + chunk_of(i, ln) * 16) : kInvalid) | dead;
        }
      };
      auto t_kstep = [&]() {
        const uint32_t k = static_cast<uint32_t>(tkb * C::BK * 2);
        tk0 = k | kmask(tkb, 0, a.K);
        tk1 = k | kmask(tkb, 1, a.K);
      };
      auto t_advance = [&]() {
        if (++tkb == nkb_g) {
          tkb = 0;
          tt += gridDim.x;
          t_setup(tt, true);
        }
        t_kstep();
      };
      auto t_load = [&](int s, int i) {  // load i < T_XL: X, else W load i - T_XL
        const uint32_t k = (i & 1) ? tk1 : tk0;
        if (i < T_XL)
          load_lds16(trs_x, t_buf(s) + wave * (16 * C::ROW) + i * 1024, (txoff[i] + k) | (k & kInvalid));
        else
          load_lds16(trs_w, t_buf(s) + T_XPART + wave * (32 * C::ROW) + (i - T_XL) * 1024,
                     (twoff[i - T_XL] + k) | (k & kInvalid));
      };
      zero_acc();
      tt = run_start;
      tkb = 0;
      t_setup(tt, false);
      t_kstep();
      // stages 0 and 1
      for (int s = 0; s < 2; ++s) {
  #pragma unroll
        for (int i = 0; i < T_LOADS; ++i) t_load(s, i);
        t_advance();
      }
      __builtin_amdgcn_s_waitcnt(wait_vm(T_LOADS));  // own stage-0 loads landed
      phase_barrier();
      int j = 0;
      for (int t = run_start; t < run_end; t += gridDim.x) {
        const TileInfo cur = tile_info(t);
        for (int kb = 0; kb < nkb_g; ++kb, ++j) {
          t_read_frags(j, 0, 0);
  #pragma unroll
          for (int ks = 0; ks < C::KSTEPS; ++ks) {
            if (ks + 1 < C::KSTEPS) t_read_frags(j, ks + 1, (ks + 1) & 1);
            // stage j + 2's six loads in the first three K-steps, two each
            constexpr int kFirst[5] = {0, 2, 4, 6, 6};
  #pragma unroll
            for (int i = kFirst[ks]; i < kFirst[ks + 1]; ++i) t_load(j + 2, i);
            t_mfma_set(ks & 1);
            __builtin_amdgcn_sched_barrier(0);
          }
          t_advance();
          __builtin_amdgcn_s_waitcnt(wait_vm(T_LOADS));  // own stage j+1 landed
          __builtin_amdgcn_s_waitcnt(kWaitLgkm0);        // this stage's LDS reads done
          phase_barrier();
        }
        // the buffer of the tile's last stage is free until the loads of the
        // stage three ahead; this wave's own W rows there are its 4 KB
        epilogue(Half<true>{}, cur, a, xrow0_t, cur.nt * OUT_COLS + wn_t * (WCOLS / 2),
                 t_buf(j - 1) + T_XPART + wave * (32 * C::ROW));
        zero_acc();
      }
    };
    run();
  };

  // ---- runs ----
  // The workgroup walks its tiles t, t + gridDim, ... in runs of one kind;
  // between runs every load has landed and every wave has passed a barrier,
  // so the next run may refill the LDS from scratch.
  // With tail tiles a run also holds tiles of one problem only (the shared
  // problem's tiles come first and are never tails), so that its loads and
  // epilogue select no problem per tile.
  for (int t = first; t < total_tiles;) {
    const bool tail = TAIL && tile_info(t).tail;
    const bool shared = PAIR && t < sp_tiles;
    int e = t;
    if constexpr (TAIL) {
      if (shared)
        e = t + ceil_div(sp_tiles - t, static_cast<int>(gridDim.x)) * static_cast<int>(gridDim.x);
      else
        while (e < total_tiles && tile_info(e).tail == tail) e += gridDim.x;
    } else {
      e = total_tiles;
    }
    run_start = t;
    run_end = e;
    if constexpr (TAIL == 1) {
      if (tail) tail_run_wide();
      else if (shared) full_run(Sel<0>{});
      else full_run(Sel<1>{});
    } else if constexpr (TAIL == 2) {
      if (tail) tail_run_half();
      else if (shared) full_run(Sel<0>{});
      else full_run(Sel<1>{});
    } else {
      full_run(Sel<-1>{});
    }
    __builtin_amdgcn_s_waitcnt(kWaitAll);
    phase_barrier();
    t = e;
  }
}

// Compute units of the current device, looked up once per device: a
// per-device cache of a fixed property (atomic, so concurrent callers are
// safe), sized for the devices one process can see.
constexpr int kMaxDevices = 64;
int device_cu_count() {
  static int cus[kMaxDevices] = {};
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  if (dev >= 0 && dev < kMaxDevices) {
    const int c = __atomic_load_n(&cus[dev], __ATOMIC_RELAXED);
    if (c > 0) return c;
  }
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) return 256;
  if (dev >= 0 && dev < kMaxDevices) __atomic_store_n(&cus[dev], n, __ATOMIC_RELAXED);
  return n;
}

template <bool GATED, int PFX, bool PAIR, bool SBLK, int TAIL>
hipError_t launch_pfx_t(const TiledArgs& ta, long long grid, hipStream_t st) {
  static unsigned long long lds_set = 0;  // devices with the LDS limit raised
  const hipError_t e_lds =
      set_max_dynamic_lds(reinterpret_cast<const void*>(&tiled_kernel<GATED, PFX, PAIR, SBLK, TAIL>),
                          Stage::LDS, &lds_set);
  if (e_lds != hipSuccess) return e_lds;
  hipLaunchKernelGGL((tiled_kernel<GATED, PFX, PAIR, SBLK, TAIL>), dim3(static_cast<unsigned>(grid)),
                     dim3(kThreads), Stage::LDS, st, ta);
  return hipGetLastError();
}

// Grouped problems (device offsets) take the kernel with tail tiles; a
// launch of static rows alone takes the blocked tile order.
template <bool GATED, int PFX>
hipError_t launch_pfx(const TiledArgs& ta, long long grid, hipStream_t st) {
  if (ta.g.offsets == nullptr) {
    if constexpr (PFX == 1) {
      if (ta.sp_tiles == 0) return launch_pfx_t<GATED, 1, false, true, 0>(ta, grid, st);
    }
    return launch_pfx_t<GATED, PFX, true, false, 0>(ta, grid, st);
  }
  // (the tail variant with 16 prefix entries per lane, for more than 256
  // groups, needs more registers than two waves per SIMD allow: there the
  // tiles stay whole)
  if constexpr (PFX > 4) {
    return launch_pfx_t<GATED, PFX, true, false, 0>(ta, grid, st);
  } else {
    // with the shared experts' tiles in the launch: half tail tiles for the
    // gated projection, whole tiles for the down projection (where tails
    // lost to the whole tiles); alone: on long K half tail tiles, which keep
    // pace with the full tiles of their weight rows, otherwise wide tail
    // tiles, fewer of them (all measured)
    if (ta.sp_tiles > 0) {
      if constexpr (GATED) return launch_pfx_t<GATED, PFX, true, false, 2>(ta, grid, st);
      else return launch_pfx_t<GATED, PFX, true, false, 0>(ta, grid, st);
    }
    if (ta.g.K >= kHalfTailK) return launch_pfx_t<GATED, PFX, false, false, 2>(ta, grid, st);
    return launch_pfx_t<GATED, PFX, false, false, 1>(ta, grid, st);
  }
}

// Host-side checks of one problem: no blocked layouts, at most kMaxGroups
// groups, and 32-bit byte offsets for a tile's X rows (all x_row_count rows
// of x when rows are indexed), a group's weight columns and a tile's output
// rows.
bool tiled_ok(const Segments& seg, const GemmArgs& a) {
  if (seg.groups > kMaxGroups || a.x_blocked || a.out_blocked) return false;
  // grouped problems: tail tiles read 2 kBN weight rows, and only a single K segment
  if (a.static_rows == 0 && a.kseg < a.K) return false;
  const size_t x_span = static_cast<size_t>(a.x_row_count > 0 ? a.x_row_count : kBM) * a.K * 2;
  const size_t w_span = (static_cast<size_t>(2 * kBN) * a.ldw +
                         (a.kseg < a.K ? static_cast<size_t>((a.K - 1) / a.kseg) * a.seg_stride : 0) + a.K) * 2;
  const size_t o_span = static_cast<size_t>(kBM + 1) * a.N * 2;
  return x_span < 0x80000000ull && w_span < 0x80000000ull && o_span < 0x80000000ull;
}

// g over seg, after sp (static rows, sp_rows of them; 0: no second problem)
template <bool GATED>
hipError_t launch_tiled_t(const Segments& seg, const GemmArgs& g, const GemmArgs& sp, int sp_rows, hipStream_t st) {
  constexpr int OUT_COLS = GATED ? kBN / 2 : kBN;
  TiledArgs ta{g, sp, 0};
  if (sp_rows > 0) ta.sp_tiles = ceil_div(sp_rows, kBM) * ceil_div(sp.N, OUT_COLS);
  const long long m_tiles = (g.offsets ? static_cast<long long>(ceil_div(seg.total_rows, kBM)) + seg.groups
                                       : ceil_div(seg.static_rows, kBM));
  const long long tiles = m_tiles * ceil_div(g.N, OUT_COLS) + ta.sp_tiles;
  if (tiles == 0) return hipSuccess;
  long long grid = std::min<long long>(tiles, device_cu_count());  // one workgroup per CU (LDS)
  grid = ((grid + 7) / 8) * 8;
  // group prefix values per lane: groups <= 64 * PFX
  if (seg.groups <= kWave) return launch_pfx<GATED, 1>(ta, grid, st);
  if (seg.groups <= 4 * kWave) return launch_pfx<GATED, 4>(ta, grid, st);
  return launch_pfx<GATED, kMaxGroups / kWave>(ta, grid, st);
}

GemmArgs up_gemm(const Segments& seg, const UpArgs& u) {
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
  return a;
}

GemmArgs down_gemm(const Segments& seg, const DownArgs& d) {
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
  return a;
}

bool up_ok(const Segments& seg, const UpArgs& u) {
  if (u.h_blocked && !ffn_streams_weights(seg)) return false;
  return !(u.x_rows && (seg.offsets == nullptr || u.x_row_count <= 0));
}

bool down_ok(const Segments& seg, const DownArgs& d) { return !(d.h_blocked && !ffn_streams_weights(seg)); }

// The limits of the kernel a problem runs on (weight streaming or tiled).
// Whether one launch takes two problems or each its own, each problem must
// pass this, and passing it is all the launchers ask.
bool gemm_ok(const Segments& seg, const GemmArgs& a) {
  return ffn_streams_weights(seg) ? skinny_ok(a) : tiled_ok(seg, a);
}

// One GEMM on its kernel, or two in one tiled launch when both take the
// tiled kernel, the second has static rows and on its own it would leave a
// partly filled last round of tiles: the routed tiles then fill it.  (When
// the shared tiles fill whole rounds the one-problem kernel is faster: the
// two-problem selections cost it about 2%.)
hipError_t launch_gemm2(const Segments& seg, const GemmArgs& a, const Segments* sh_seg, const GemmArgs* sh,
                        bool gated, hipStream_t st) {
  const bool tiled = !ffn_streams_weights(seg);
  const int out_cols = gated ? kBN / 2 : kBN;
  const bool merge = sh != nullptr && tiled && !ffn_streams_weights(*sh_seg) && sh_seg->offsets == nullptr &&
                     static_cast<long long>(ceil_div(sh_seg->static_rows, kBM)) * ceil_div(sh->N, out_cols) %
                             device_cu_count() != 0;
  if (merge) {
    if (!tiled_ok(seg, a) || !tiled_ok(*sh_seg, *sh)) return hipErrorInvalidValue;
    return gated ? launch_tiled_t<true>(seg, a, *sh, sh_seg->static_rows, st)
                 : launch_tiled_t<false>(seg, a, *sh, sh_seg->static_rows, st);
  }
  hipError_t e = tiled ? launch_tiled(seg, a, gated, st) : launch_skinny(seg, a, gated, st);
  if (e != hipSuccess || sh == nullptr) return e;
  return ffn_streams_weights(*sh_seg) ? launch_skinny(*sh_seg, *sh, gated, st) : launch_tiled(*sh_seg, *sh, gated, st);
}

}  // namespace

hipError_t launch_tiled(const Segments& seg, const GemmArgs& a, bool gated, hipStream_t st) {
  if (!tiled_ok(seg, a)) return hipErrorInvalidValue;
  const GemmArgs none{};
  return gated ? launch_tiled_t<true>(seg, a, none, 0, st) : launch_tiled_t<false>(seg, a, none, 0, st);
}

bool ffn_streams_weights(const Segments& seg) { return seg.max_rows <= kSkinnyMaxRows; }

bool ffn_up_supported(const Segments& seg, const UpArgs& u) { return up_ok(seg, u) && gemm_ok(seg, up_gemm(seg, u)); }

bool ffn_down_supported(const Segments& seg, const DownArgs& d) {
  return down_ok(seg, d) && gemm_ok(seg, down_gemm(seg, d));
}

hipError_t launch_ffn_up(const Segments& seg, const UpArgs& u, hipStream_t st) {
  if (!up_ok(seg, u)) return hipErrorInvalidValue;
  return launch_gemm2(seg, up_gemm(seg, u), nullptr, nullptr, true, st);
}

hipError_t launch_ffn_up2(const Segments& seg, const UpArgs& u, const Segments& sh_seg, const UpArgs& sh,
                          hipStream_t st) {
  if (!up_ok(seg, u) || !up_ok(sh_seg, sh)) return hipErrorInvalidValue;
  const GemmArgs s = up_gemm(sh_seg, sh);
  return launch_gemm2(seg, up_gemm(seg, u), &sh_seg, &s, true, st);
}

hipError_t launch_ffn_down(const Segments& seg, const DownArgs& d, hipStream_t st) {
  if (!down_ok(seg, d)) return hipErrorInvalidValue;
  return launch_gemm2(seg, down_gemm(seg, d), nullptr, nullptr, false, st);
}

hipError_t launch_ffn_down2(const Segments& seg, const DownArgs& d, const Segments& sh_seg, const DownArgs& sh,
                            hipStream_t st) {
  if (!down_ok(seg, d) || !down_ok(sh_seg, sh)) return hipErrorInvalidValue;
  const GemmArgs s = down_gemm(sh_seg, sh);
  return launch_gemm2(seg, down_gemm(seg, d), &sh_seg, &s, false, st);
}

}  // namespace moe
