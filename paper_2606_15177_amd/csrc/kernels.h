// Host-side launchers of the gfx950 kernels; the C ABI composes them.
// Every launcher only enqueues work on `st` and returns hipGetLastError().
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace moe {

// ---- route.hip -------------------------------------------------------------
// Gating variant of the router (see moe.h): gate 0 softmax over the picks,
// 1 full softmax, 2 sigmoid scores; bias (selection only, gate 2), scale,
// and a group limit when n_group > 1 (n_group <= 64).
struct RouteGating {
  int gate;
  const float* bias;
  float scale;
  int n_group, topk_group;
};
// The dispatch outputs of launch_permute (offsets, perm_token, inv_pos) for
// the local slots of local_experts (nullptr: slot = expert id).
struct DispatchArgs {
  const int32_t* local_experts;
  int E_local;
  int32_t* offsets;
  int32_t* perm_token;
  int32_t* inv_pos;
};
// Batches of at most this many (token, expert) pairs are dispatched by one block.
constexpr int kDispatchPairs = 512;
// Experts per layer (E, and so E_local) that the kernels take.
constexpr int kMaxExperts = 1024;

// Top-k selection + gates; when counts != nullptr also accumulates the
// source x expert counts (and sets expert_load if non-null, which must have
// been zeroed on the stream before).  gating == nullptr: softmax over the
// picks, unscaled, no group limit.  dispatch (nullable): when the batch is
// small enough for one block to route it (decode-sized batches), that block
// also writes the dispatch, exactly as launch_permute would; *dispatched
// says whether it did (the caller then skips launch_permute).
hipError_t launch_route(int T, int E, int k, const float* logits, int32_t* topk_idx,
                        float* topk_w, const int32_t* src, int S, int64_t* counts,
                        int32_t* expert_load, const RouteGating* gating, hipStream_t st,
                        const DispatchArgs* dispatch = nullptr, bool* dispatched = nullptr);
// Counts from (src, topk_idx); expert_load as above.
hipError_t launch_route_stats(int T, int k, int S, int E, const int32_t* src,
                              const int32_t* topk_idx, int64_t* counts, int32_t* expert_load,
                              hipStream_t st);
hipError_t launch_fill_i32(int32_t* p, int n, int32_t value, hipStream_t st);

// ---- permute.hip -----------------------------------------------------------
// Workspace of launch_permute; with S and E (the statistics' shape) it also
// holds the count pass's per-tile histograms where those are summed in two
// levels, and a call with counts needs the size for its S and E.
size_t permute_ws_bytes(int T, int k, int E_local, int S = 0, int E = 0);
// offsets / perm_token / inv_pos of the stable dispatch sort.  With counts
// != nullptr the launches also accumulate the source x expert counts of all
// T*k pairs (and add to expert_load as launch_route does); only for
// T*k > kDispatchPairs, where that pass runs (else hipErrorInvalidValue).
hipError_t launch_permute(int T, int k, int E, int E_local, const int32_t* local_experts,
                          const int32_t* topk_idx, int32_t* offsets, int32_t* perm_token,
                          int32_t* inv_pos, void* ws, hipStream_t st, const int32_t* src = nullptr,
                          int S = 0, int64_t* counts = nullptr, int32_t* expert_load = nullptr);
// x_perm[r] = x[perm_token[r]] for r < *n_rows (device scalar), capacity rows.
hipError_t launch_gather_rows(int capacity, int H, const int32_t* perm_token,
                              const int32_t* n_rows, const uint16_t* x, uint16_t* x_perm,
                              hipStream_t st);

// ---- ffn_*.hip -------------------------------------------------------------
// A grouped GEMM over row segments.  Group g owns rows [offsets[g],
// offsets[g+1]) of the activation matrix (or rows [0, static_rows) of a single
// group when offsets == nullptr).  max_rows bounds the rows of any one group
// and total_rows the rows of all groups (both host-side capacities).
struct Segments {
  const int32_t* offsets;
  int groups;
  int static_rows;
  int max_rows;
  int total_rows;
};

// h[r][i] = silu(sum_c X[r][c] Wg[g][i][c]) * (sum_c X[r][c] Wu[g][i][c]),
// weights [groups][N][K] (group stride N*K), x row stride K, h row stride N.
// X[r] = x[r], or x[x_rows[r]] when x_rows != nullptr (the dispatch gather
// read in place; x then has x_row_count rows; x_row_count is 0 otherwise).
struct UpArgs {
  const uint16_t* x;
  const uint16_t* w_gate;
  const uint16_t* w_up;
  uint16_t* h;
  int K, N;
  const int32_t* x_rows;
  int x_row_count;
  // write h in the chunk-blocked layout (decode-sized groups, see below)
  bool h_blocked;
};
hipError_t launch_ffn_up(const Segments& seg, const UpArgs& a, hipStream_t st);
// Host only, no HIP call: whether launch_ffn_up accepts these sizes (the
// pointers are not looked at; x_row_count > 0 stands for rows read through
// x_rows).  launch_ffn_up2 accepts two problems when each passes.
bool ffn_up_supported(const Segments& seg, const UpArgs& a);
// The same for the routed experts (seg, a) and the shared experts (sh_seg
// with static rows, sh): one launch when both take the tiled kernel, the
// shared tiles first.
hipError_t launch_ffn_up2(const Segments& seg, const UpArgs& a, const Segments& sh_seg, const UpArgs& sh,
                          hipStream_t st);
// True when these segments take the weight-streaming kernels (decode-sized
// groups).
bool ffn_streams_weights(const Segments& seg);

// For decode-sized groups (ffn_streams_weights) the gate/up GEMM may write h
// chunk-blocked: each group's rows cut into chunks of 32 (the last one
// zero-padded) whose 1 KB blocks are MFMA operand fragments, which the down
// GEMM then loads as whole contiguous kilobytes.  Such an h holds
// chunk_capacity(groups, total_rows) chunks of 32 x N; N and the down GEMM's
// K must be multiples of 16.
size_t chunk_capacity(int groups, int total_rows);
constexpr int kChunkRowsHost = 32;  // rows of a chunk of the blocked layout

// y[r][n] = sum_c h[r][c] Wd(g, n, c), h row stride K, y row stride N.
// Wd(g, n, c) = w[g*group_stride + (c / kseg)*seg_stride + n*ldw + c % kseg]
// (one segment per group for routed experts; the stacked shared experts use
// kseg = I_shared so that the K range runs over all of them).
struct DownArgs {
  const uint16_t* h;
  const uint16_t* w;
  uint16_t* y;
  int K, N, kseg, ldw;
  size_t seg_stride, group_stride;
  // h in the chunk-blocked layout written by launch_ffn_up
  bool h_blocked;
};
hipError_t launch_ffn_down(const Segments& seg, const DownArgs& a, hipStream_t st);
// Host only: whether launch_ffn_down accepts these sizes (as above).
bool ffn_down_supported(const Segments& seg, const DownArgs& a);
hipError_t launch_ffn_down2(const Segments& seg, const DownArgs& a, const Segments& sh_seg, const DownArgs& sh,
                            hipStream_t st);

// ---- combine.hip -----------------------------------------------------------
hipError_t launch_combine(int T, int k, int H, const uint16_t* y_perm, const int32_t* inv_pos,
                          const float* topk_w, const uint16_t* y_shared, uint16_t* out,
                          hipStream_t st);

// ---- place.hip -------------------------------------------------------------
// Source-aware expert placement, one workgroup per layer (see moe.h).
constexpr int kPlaceMaxExperts = 1024;
constexpr int kPlaceMaxRanks = 64;           // ranks are the lanes of one wave
constexpr int kPlaceMaxSourceRanks = 4096;   // S*G entries of D staged in LDS
constexpr int kPlaceMaxLdsBytes = 160 * 1024;
struct PlaceArgs {
  int L, S, E, G;
  int slots;  // row length of rank_experts
  double alpha, beta, gamma, m_uniform;
  const int32_t* cap;  // host [G]
  const int64_t* A;    // [L][S][E]
  const int64_t* B;    // [L][E] or null
  const double* D;     // [S][G]
  const double* M;     // [L][E][G] or null
  const int32_t* x0;   // [L][E]
  int32_t* x;          // [L][E]
  int32_t* rank_experts;  // [L][G][slots] or null
  double* cost;           // [L][3] or null
};
size_t place_lds_bytes(int S, int E, int G);
hipError_t launch_place(const PlaceArgs& a, hipStream_t st);

// ---- window.hip ------------------------------------------------------------
// Window diagnostics under a placement (see moe.h).
constexpr int kWindowMaxExperts = 8192;
constexpr int kWindowMaxRanks = 1024;
constexpr int kWindowMaxEngines = 1024;
struct WindowArgs {
  int L, S, E, G, n_engines;
  const int64_t* A;       // [L][S][E]
  const int64_t* B;       // [L][E] or null
  const int32_t* x;       // [L][E]
  const int32_t* home;    // [S]
  const int32_t* engine;  // [G] or null (rank g is engine g)
  int64_t* remote;        // [L][S]
  int64_t* total;         // [L][S]
  int64_t* rank_load;     // [L][G]
  double* pressure;       // [n_engines] or null
};
hipError_t launch_window(const WindowArgs& a, hipStream_t st);

}  // namespace moe
