// The C ABI (include/moe.h): host-side validation, workspace carving and the
// launch sequence of each entry point.  No allocation, no synchronisation,
// no device-to-host traffic: every data-dependent size stays on the device.
#include "moe.h"

#include <algorithm>

#include "kernels.h"

namespace {

constexpr size_t kAlign = 256;
constexpr int64_t kIntMax = 2147483647;

size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int check_dims(const moe_dims* d) {
  if (d == nullptr) return MOE_ERR_NULL;
  if (d->T < 0 || d->H < 1 || d->E < 1 || d->k < 1 || d->k > d->E || d->I < 1 || d->S < 1 ||
      d->E_local < 1 || d->E_local > d->E || d->n_shared < 0 ||
      (d->n_shared > 0 && d->I_shared < 1))
    return MOE_ERR_DIMS;
  if (d->flags < MOE_GATE_SOFTMAX_TOPK || d->flags > MOE_GATE_SIGMOID) return MOE_ERR_UNSUPPORTED;
  if (d->E > moe::kMaxExperts || d->k > 32) return MOE_ERR_UNSUPPORTED;
  if (d->H % 8 != 0 || d->I % 8 != 0 || (d->n_shared > 0 && d->I_shared % 8 != 0))
    return MOE_ERR_UNSUPPORTED;
  if (static_cast<int64_t>(d->T) * d->k > kIntMax || static_cast<int64_t>(d->S) * d->E > kIntMax ||
      static_cast<int64_t>(d->n_shared) * std::max(d->I_shared, 0) > kIntMax)
    return MOE_ERR_UNSUPPORTED;
  return MOE_OK;
}

// The router's gating variant: dims->flags picks the gate function, g (may be
// null) carries its parameters.
int gating_ok(const moe_dims* d, const moe_gating* g, moe::RouteGating* out) {
  *out = moe::RouteGating{d->flags, nullptr, 1.0f, 0, 0};
  if (g == nullptr) return MOE_OK;
  if (g->bias && d->flags != MOE_GATE_SIGMOID) return MOE_ERR_DIMS;
  if (g->bias && (reinterpret_cast<uintptr_t>(g->bias) & 3u) != 0) return MOE_ERR_ALIGN;
  if (g->n_group > 1) {
    if (g->n_group > 64) return MOE_ERR_UNSUPPORTED;
    if (d->E % g->n_group != 0 || g->topk_group < 1 || g->topk_group > g->n_group ||
        d->k > g->topk_group * (d->E / g->n_group))
      return MOE_ERR_DIMS;
  } else if (g->n_group < 0) {
    return MOE_ERR_DIMS;
  }
  *out = moe::RouteGating{d->flags, g->bias, g->routed_scale, g->n_group, g->topk_group};
  return MOE_OK;
}

int64_t sh_width(const moe_dims* d) {
  return d->n_shared > 0 ? static_cast<int64_t>(d->n_shared) * d->I_shared : 0;
}

// Decode-sized batches run the routed GEMMs on chunk-blocked activations.
bool ffn_blocked(const moe_dims* d) {
  const moe::Segments routed{nullptr, d->E_local, 0, d->T, d->T * d->k};
  return d->T > 0 && moe::ffn_streams_weights(routed) && d->H % 16 == 0 && d->I % 16 == 0;
}

// Workspace of the expert FFN: h (chunk-blocked for decode-sized batches),
// then h_shared.
struct FfnWs {
  uint16_t* h;
  bool h_blocked;
  uint16_t* h_sh;
  size_t bytes;
};
FfnWs carve_ffn(const moe_dims* d, void* base) {
  FfnWs w{};
  unsigned char* p = static_cast<unsigned char*>(base);
  size_t off = 0;
  auto take = [&](size_t bytes) {
    unsigned char* r = p ? p + off : nullptr;
    off += align_up(bytes);
    return r;
  };
  const size_t rows = static_cast<size_t>(d->T) * d->k;
  w.h_blocked = ffn_blocked(d);
  if (w.h_blocked) {
    const size_t chunk_rows = moe::chunk_capacity(d->E_local, static_cast<int>(rows)) * moe::kChunkRowsHost;
    w.h = reinterpret_cast<uint16_t*>(take(chunk_rows * d->I * sizeof(uint16_t)));
  } else {
    w.h = reinterpret_cast<uint16_t*>(take(rows * d->I * sizeof(uint16_t)));
  }
  w.h_sh = reinterpret_cast<uint16_t*>(take(static_cast<size_t>(d->T) * sh_width(d) * sizeof(uint16_t)));
  w.bytes = off;
  return w;
}
size_t ffn_ws(const moe_dims* d) { return carve_ffn(d, nullptr).bytes; }

// The forward workspace, carved in this order.
struct ForwardWs {
  int32_t* topk_idx;
  float* topk_w;
  int32_t* offsets;
  int32_t* perm_token;
  int32_t* inv_pos;
  uint16_t* y_perm;
  uint16_t* y_shared;
  void* permute_ws;
  void* ffn_ws;
  size_t bytes;
};

ForwardWs carve_forward(const moe_dims* d, void* base) {
  ForwardWs w{};
  unsigned char* p = static_cast<unsigned char*>(base);
  size_t off = 0;
  auto take = [&](size_t bytes) {
    unsigned char* r = p ? p + off : nullptr;
    off += align_up(bytes);
    return r;
  };
  const size_t rows = static_cast<size_t>(d->T) * d->k;
  w.topk_idx = reinterpret_cast<int32_t*>(take(rows * sizeof(int32_t)));
  w.topk_w = reinterpret_cast<float*>(take(rows * sizeof(float)));
  w.offsets = reinterpret_cast<int32_t*>(take((d->E_local + 1) * sizeof(int32_t)));
  w.perm_token = reinterpret_cast<int32_t*>(take(rows * sizeof(int32_t)));
  w.inv_pos = reinterpret_cast<int32_t*>(take(rows * sizeof(int32_t)));
  w.y_perm = reinterpret_cast<uint16_t*>(take(rows * d->H * sizeof(uint16_t)));
  w.y_shared = reinterpret_cast<uint16_t*>(
      take(d->n_shared > 0 ? static_cast<size_t>(d->T) * d->H * sizeof(uint16_t) : 0));
  w.permute_ws = take(moe::permute_ws_bytes(d->T, d->k, d->E_local, d->S, d->E));
  w.ffn_ws = take(ffn_ws(d));
  w.bytes = off;
  return w;
}

size_t entry_ws(const moe_dims* d, int entry) {
  switch (entry) {
    case MOE_ENTRY_PERMUTE:
      return align_up(moe::permute_ws_bytes(d->T, d->k, d->E_local));
    case MOE_ENTRY_EXPERT_FFN:
      return ffn_ws(d);
    case MOE_ENTRY_FORWARD:
      return carve_forward(d, nullptr).bytes;
    default:
      return 0;
  }
}

int check_ws(const moe_dims* d, int entry, const void* ws, size_t ws_bytes) {
  const size_t need = entry_ws(d, entry);
  if (ws_bytes < need) return MOE_ERR_WORKSPACE;
  if (need > 0 && ws == nullptr) return MOE_ERR_WORKSPACE;
  if (ws != nullptr && (reinterpret_cast<uintptr_t>(ws) % kAlign) != 0) return MOE_ERR_ALIGN;
  return MOE_OK;
}

int status(hipError_t e) { return e == hipSuccess ? MOE_OK : MOE_ERR_DEVICE; }

void record(const moe_taps* taps, int slot, hipStream_t st) {
  if (taps && taps->events[slot]) (void)hipEventRecord(static_cast<hipEvent_t>(taps->events[slot]), st);
}

int weights_ok(const moe_dims* d, const moe_weights* w) {
  if (w == nullptr || w->w_gate == nullptr || w->w_up == nullptr || w->w_down == nullptr)
    return MOE_ERR_NULL;
  if (d->n_shared > 0 && (w->sh_gate == nullptr || w->sh_up == nullptr || w->sh_down == nullptr))
    return MOE_ERR_NULL;
  if (!aligned16(w->w_gate) || !aligned16(w->w_up) || !aligned16(w->w_down)) return MOE_ERR_ALIGN;
  if (d->n_shared > 0 && (!aligned16(w->sh_gate) || !aligned16(w->sh_up) || !aligned16(w->sh_down)))
    return MOE_ERR_ALIGN;
  return MOE_OK;
}

// The two grouped GEMMs of the experts (routed, then shared): their row
// segments and arguments, built the same way for the host-side limit check
// (null pointers; rows_indexed says whether the gate/up GEMM reads its rows
// through a row list of T entries) and for the launches.
struct FfnPlan {
  moe::Segments routed, shared;
  moe::UpArgs up, sh_up;
  moe::DownArgs dn, sh_dn;
};
FfnPlan plan_ffn(const moe_dims* d, const uint16_t* x_perm, const int32_t* x_rows, bool rows_indexed,
                 const int32_t* offsets, const moe_weights* w, const uint16_t* x, uint16_t* y_perm,
                 uint16_t* y_shared, void* ws) {
  const FfnWs fw = carve_ffn(d, ws);
  const int shw = static_cast<int>(sh_width(d));
  FfnPlan p{};
  p.routed = moe::Segments{offsets, d->E_local, 0, d->T, d->T * d->k};
  p.shared = moe::Segments{nullptr, 1, d->T, d->T, d->T};
  p.up = moe::UpArgs{x_perm, w ? w->w_gate : nullptr, w ? w->w_up : nullptr, fw.h, d->H, d->I, x_rows,
                     rows_indexed ? d->T : 0, fw.h_blocked};
  p.sh_up = moe::UpArgs{x, w ? w->sh_gate : nullptr, w ? w->sh_up : nullptr, fw.h_sh, d->H, shw, nullptr, 0, false};
  p.dn = moe::DownArgs{fw.h, w ? w->w_down : nullptr, y_perm, d->I, d->H, d->I, d->I, 0,
                       static_cast<size_t>(d->H) * d->I, fw.h_blocked};
  p.sh_dn = moe::DownArgs{fw.h_sh, w ? w->sh_down : nullptr, y_shared, shw, d->H, d->I_shared, d->I_shared,
                          static_cast<size_t>(d->H) * d->I_shared, 0, false};
  return p;
}

// Kernel limits of the expert GEMMs for these sizes (MOE_ERR_UNSUPPORTED
// beyond them), decided before anything is enqueued: the same predicates the
// launchers apply, on the same arguments.
int check_ffn_limits(const moe_dims* d, bool rows_indexed) {
  if (d->T == 0) return MOE_OK;
  const FfnPlan p = plan_ffn(d, nullptr, nullptr, rows_indexed, nullptr, nullptr, nullptr, nullptr, nullptr,
                             nullptr);
  if (!moe::ffn_up_supported(p.routed, p.up) || !moe::ffn_down_supported(p.routed, p.dn))
    return MOE_ERR_UNSUPPORTED;
  if (d->n_shared > 0 &&
      (!moe::ffn_up_supported(p.shared, p.sh_up) || !moe::ffn_down_supported(p.shared, p.sh_dn)))
    return MOE_ERR_UNSUPPORTED;
  return MOE_OK;
}

// The limits of one entry point (0: of every entry point).
int check_entry(const moe_dims* d, int entry) {
  int s = MOE_OK;
  if (entry == 0 || entry == MOE_ENTRY_EXPERT_FFN) s = check_ffn_limits(d, false);
  if (s == MOE_OK && (entry == 0 || entry == MOE_ENTRY_FORWARD)) s = check_ffn_limits(d, true);
  return s;
}

int run_ffn(const moe_dims* d, const uint16_t* x_perm, const int32_t* x_rows, const int32_t* offsets,
            const moe_weights* w, const uint16_t* x, uint16_t* y_perm, uint16_t* y_shared,
            void* ws, const moe_taps* taps, hipStream_t st) {
  const FfnPlan p = plan_ffn(d, x_perm, x_rows, x_rows != nullptr, offsets, w, x, y_perm, y_shared, ws);
  hipError_t e;

  // routed and shared experts: one launch per GEMM when both take the tiled
  // kernel, else one each
  record(taps, 2 * MOE_STAGE_FFN_UP, st);
  if (d->n_shared > 0)
    e = moe::launch_ffn_up2(p.routed, p.up, p.shared, p.sh_up, st);
  else
    e = moe::launch_ffn_up(p.routed, p.up, st);
  if (e != hipSuccess) return MOE_ERR_DEVICE;
  record(taps, 2 * MOE_STAGE_FFN_UP + 1, st);

  record(taps, 2 * MOE_STAGE_FFN_DOWN, st);
  if (d->n_shared > 0)
    e = moe::launch_ffn_down2(p.routed, p.dn, p.shared, p.sh_dn, st);
  else
    e = moe::launch_ffn_down(p.routed, p.dn, st);
  if (e != hipSuccess) return MOE_ERR_DEVICE;
  record(taps, 2 * MOE_STAGE_FFN_DOWN + 1, st);
  return MOE_OK;
}

// The workspace of moe_forward_noalloc: a library-owned device array, one
// copy per device (every device the library runs on holds it until the
// process ends).  Host code never uses its name as an address: the address
// of a device's copy comes from hipGetSymbolAddress on that device.
static __device__ __align__(256) unsigned char scratch[MOE_NOALLOC_SCRATCH_BYTES];

// The device address of the current device's copy of `scratch`, looked up
// once per device (the pointers are cached with atomic operations, so
// concurrent first calls are safe); nullptr when the lookup fails.
void* scratch_address() {
  constexpr int kMaxDevices = 64;
  static void* addr[kMaxDevices] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  void* p = __atomic_load_n(&addr[dev], __ATOMIC_ACQUIRE);
  if (p != nullptr) return p;
  if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) {
    (void)hipGetLastError();
    return nullptr;
  }
  __atomic_store_n(&addr[dev], p, __ATOMIC_RELEASE);
  return p;
}

}  // namespace

extern "C" {

int moe_abi_version(void) { return MOE_ABI_VERSION; }

const char* moe_strerror(int s) {
  switch (s) {
    case MOE_OK: return "ok";
    case MOE_ERR_NULL: return "a required pointer is NULL";
    case MOE_ERR_DIMS: return "inconsistent or negative dimensions";
    case MOE_ERR_UNSUPPORTED: return "dimensions beyond the kernels' limits";
    case MOE_ERR_WORKSPACE: return "workspace missing or too small";
    case MOE_ERR_DEVICE: return "kernel launch failed";
    case MOE_ERR_ALIGN: return "pointer not aligned as required";
    default: return "unknown status";
  }
}

size_t moe_workspace_bytes(const moe_dims* d, int entry) {
  if (check_dims(d) != MOE_OK || check_entry(d, entry) != MOE_OK) return 0;
  return entry_ws(d, entry);
}

int moe_validate(const moe_dims* d, int entry, size_t ws_bytes) {
  int s = check_dims(d);
  if (s != MOE_OK) return s;
  s = check_entry(d, entry);
  if (s != MOE_OK) return s;
  if (entry != 0 && ws_bytes < entry_ws(d, entry)) return MOE_ERR_WORKSPACE;
  return MOE_OK;
}

int moe_route(const moe_dims* d, const moe_gating* gating, const float* logits, int32_t* topk_idx,
              float* topk_w, void* stream) {
  int s = check_dims(d);
  if (s != MOE_OK) return s;
  moe::RouteGating rg;
  s = gating_ok(d, gating, &rg);
  if (s != MOE_OK) return s;
  if (d->T > 0 && (!logits || !topk_idx || !topk_w)) return MOE_ERR_NULL;
  return status(moe::launch_route(d->T, d->E, d->k, logits, topk_idx, topk_w, nullptr, d->S,
                                  nullptr, nullptr, &rg, static_cast<hipStream_t>(stream)));
}

int moe_route_stats(const moe_dims* d, const int32_t* src, const int32_t* topk_idx,
                    int64_t* counts, int32_t* expert_load, void* stream) {
  int s = check_dims(d);
  if (s != MOE_OK) return s;
  if (!counts || (d->T > 0 && (!src || !topk_idx))) return MOE_ERR_NULL;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (expert_load && moe::launch_fill_i32(expert_load, d->E, 0, st) != hipSuccess)
    return MOE_ERR_DEVICE;
  return status(moe::launch_route_stats(d->T, d->k, d->S, d->E, src, topk_idx, counts,
                                        expert_load, st));
}

int moe_permute(const moe_dims* d, const int32_t* topk_idx, const int32_t* local_experts,
                const moe_bf16* x, int32_t* offsets, int32_t* perm_token, int32_t* inv_pos,
                moe_bf16* x_perm, void* ws, size_t ws_bytes, void* stream) {
  int s = check_dims(d);
  if (s != MOE_OK) return s;
  if (!local_experts && d->E_local != d->E) return MOE_ERR_DIMS;
  if (!offsets || (d->T > 0 && (!topk_idx || !perm_token || !inv_pos))) return MOE_ERR_NULL;
  if ((x == nullptr) != (x_perm == nullptr)) return MOE_ERR_NULL;
  if (x && (!aligned16(x) || !aligned16(x_perm))) return MOE_ERR_ALIGN;
  s = check_ws(d, MOE_ENTRY_PERMUTE, ws, ws_bytes);
  if (s != MOE_OK) return s;
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipError_t e = moe::launch_permute(d->T, d->k, d->E, d->E_local, local_experts, topk_idx,
                                     offsets, perm_token, inv_pos, ws, st);
  if (e != hipSuccess) return MOE_ERR_DEVICE;
  if (x) {
    e = moe::launch_gather_rows(d->T * d->k, d->H, perm_token, offsets + d->E_local, x, x_perm, st);
    if (e != hipSuccess) return MOE_ERR_DEVICE;
  }
  return MOE_OK;
}

int moe_expert_ffn(const moe_dims* d, const moe_bf16* x_perm, const int32_t* offsets,
                   const moe_weights* w, const moe_bf16* x, moe_bf16* y_perm, moe_bf16* y_shared,
                   void* ws, size_t ws_bytes, void* stream) {
  int s = check_dims(d);
  if (s != MOE_OK) return s;
  s = weights_ok(d, w);
  if (s != MOE_OK) return s;
  if (!x_perm || !offsets || !y_perm) return MOE_ERR_NULL;
  if (d->n_shared > 0 && (!x || !y_shared)) return MOE_ERR_NULL;
  if (!aligned16(x_perm) || !aligned16(y_perm)) return MOE_ERR_ALIGN;
  if (d->n_shared > 0 && (!aligned16(x) || !aligned16(y_shared))) return MOE_ERR_ALIGN;
  s = check_entry(d, MOE_ENTRY_EXPERT_FFN);
  if (s != MOE_OK) return s;
  s = check_ws(d, MOE_ENTRY_EXPERT_FFN, ws, ws_bytes);
  if (s != MOE_OK) return s;
  if (d->T == 0) return MOE_OK;
  return run_ffn(d, x_perm, nullptr, offsets, w, x, y_perm, y_shared, ws, nullptr,
                 static_cast<hipStream_t>(stream));
}

int moe_combine(const moe_dims* d, const moe_bf16* y_perm, const int32_t* inv_pos,
                const float* topk_w, const moe_bf16* y_shared, moe_bf16* out, void* stream) {
  int s = check_dims(d);
  if (s != MOE_OK) return s;
  if (d->T > 0 && (!y_perm || !inv_pos || !topk_w || !out)) return MOE_ERR_NULL;
  if (d->T > 0 && (!aligned16(y_perm) || !aligned16(out) || (y_shared && !aligned16(y_shared))))
    return MOE_ERR_ALIGN;
  return status(moe::launch_combine(d->T, d->k, d->H, y_perm, inv_pos, topk_w, y_shared, out,
                                    static_cast<hipStream_t>(stream)));
}

int moe_forward(const moe_dims* d, const moe_gating* gating, const float* logits, const int32_t* src,
                const moe_bf16* x, const int32_t* local_experts, const moe_weights* w, int64_t* counts,
                moe_bf16* out, const moe_taps* taps, void* ws, size_t ws_bytes, void* stream) {
  int s = check_dims(d);
  if (s != MOE_OK) return s;
  moe::RouteGating rg;
  s = gating_ok(d, gating, &rg);
  if (s != MOE_OK) return s;
  if (!local_experts && d->E_local != d->E) return MOE_ERR_DIMS;
  s = weights_ok(d, w);
  if (s != MOE_OK) return s;
  if (d->T > 0 && (!logits || !x || !out)) return MOE_ERR_NULL;
  if (counts && d->T > 0 && !src) return MOE_ERR_NULL;
  if (d->T > 0 && (!aligned16(x) || !aligned16(out))) return MOE_ERR_ALIGN;
  s = check_entry(d, MOE_ENTRY_FORWARD);
  if (s != MOE_OK) return s;
  s = check_ws(d, MOE_ENTRY_FORWARD, ws, ws_bytes);
  if (s != MOE_OK) return s;

  hipStream_t st = static_cast<hipStream_t>(stream);
  ForwardWs fw = carve_forward(d, ws);
  int32_t* topk_idx = (taps && taps->topk_idx) ? taps->topk_idx : fw.topk_idx;
  float* topk_w = (taps && taps->topk_w) ? taps->topk_w : fw.topk_w;
  int32_t* offsets = (taps && taps->offsets) ? taps->offsets : fw.offsets;
  int32_t* perm_token = (taps && taps->perm_token) ? taps->perm_token : fw.perm_token;
  int32_t* inv_pos = (taps && taps->inv_pos) ? taps->inv_pos : fw.inv_pos;
  int32_t* expert_load = taps ? taps->expert_load : nullptr;
  hipError_t e;

  record(taps, 2 * MOE_STAGE_ROUTE, st);
  if (counts && expert_load) {
    e = moe::launch_fill_i32(expert_load, d->E, 0, st);
    if (e != hipSuccess) return MOE_ERR_DEVICE;
  }
  // decode-sized batches: the routing launch also writes the dispatch.
  // Larger ones are dispatched by the permute passes, whose count pass then
  // also takes the statistics: its blocks hold many more pairs than the
  // router's, and their histograms are summed in two levels (see
  // permute.hip) rather than by global atomics per bin and block.
  const moe::DispatchArgs disp{local_experts, d->E_local, offsets, perm_token, inv_pos};
  const bool stats_in_permute = counts != nullptr && static_cast<int64_t>(d->T) * d->k > moe::kDispatchPairs;
  int64_t* route_counts = stats_in_permute ? nullptr : counts;
  bool dispatched = false;
  e = moe::launch_route(d->T, d->E, d->k, logits, topk_idx, topk_w, route_counts ? src : nullptr, d->S,
                        route_counts, route_counts ? expert_load : nullptr, &rg, st, &disp, &dispatched);
  if (e != hipSuccess) return MOE_ERR_DEVICE;
  record(taps, 2 * MOE_STAGE_ROUTE + 1, st);

  record(taps, 2 * MOE_STAGE_PERMUTE, st);
  if (!dispatched) {
    e = moe::launch_permute(d->T, d->k, d->E, d->E_local, local_experts, topk_idx, offsets, perm_token,
                            inv_pos, fw.permute_ws, st, src, d->S, stats_in_permute ? counts : nullptr,
                            stats_in_permute ? expert_load : nullptr);
    if (e != hipSuccess) return MOE_ERR_DEVICE;
  }
  // no gathered copy of x: the gate/up GEMM reads its rows through perm_token
  record(taps, 2 * MOE_STAGE_PERMUTE + 1, st);

  if (d->T > 0) {
    s = run_ffn(d, x, perm_token, offsets, w, x, fw.y_perm, fw.y_shared, fw.ffn_ws, taps, st);
    if (s != MOE_OK) return s;
  } else {
    record(taps, 2 * MOE_STAGE_FFN_UP, st);
    record(taps, 2 * MOE_STAGE_FFN_UP + 1, st);
    record(taps, 2 * MOE_STAGE_FFN_DOWN, st);
    record(taps, 2 * MOE_STAGE_FFN_DOWN + 1, st);
  }

  record(taps, 2 * MOE_STAGE_COMBINE, st);
  e = moe::launch_combine(d->T, d->k, d->H, fw.y_perm, inv_pos, topk_w,
                          d->n_shared > 0 ? fw.y_shared : nullptr, out, st);
  if (e != hipSuccess) return MOE_ERR_DEVICE;
  record(taps, 2 * MOE_STAGE_COMBINE + 1, st);
  return MOE_OK;
}

int moe_forward_noalloc(const moe_dims* d, const moe_gating* gating, const float* logits, const int32_t* src,
                        const moe_bf16* x, const int32_t* local_experts, const moe_weights* w, int64_t* counts,
                        moe_bf16* out, const moe_taps* taps, void* stream) {
  int s = check_dims(d);
  if (s != MOE_OK) return s;
  s = check_entry(d, MOE_ENTRY_FORWARD);
  if (s != MOE_OK) return s;
  if (entry_ws(d, MOE_ENTRY_FORWARD) > MOE_NOALLOC_SCRATCH_BYTES) return MOE_ERR_WORKSPACE;
  // the scratch copy used is the current device's: the stream must be one of its streams
  int cur = 0, sdev = 0;
  if (hipGetDevice(&cur) != hipSuccess || hipStreamGetDevice(static_cast<hipStream_t>(stream), &sdev) != hipSuccess ||
      cur != sdev)
    return MOE_ERR_DEVICE;
  void* ws = scratch_address();
  if (ws == nullptr) return MOE_ERR_DEVICE;
  // the forward workspace needs no initialisation: every region is written
  // before it is read within the call
  return moe_forward(d, gating, logits, src, x, local_experts, w, counts, out, taps, ws,
                     MOE_NOALLOC_SCRATCH_BYTES, stream);
}

size_t moe_place_slots(const moe_place_dims* pd, const int32_t* cap) {
  if (pd == nullptr || cap == nullptr || pd->E < 1 || pd->G < 1) return 0;
  int slots = 0;
  for (int g = 0; g < pd->G; ++g) slots = std::max(slots, std::min(std::max(cap[g], 0), pd->E));
  return static_cast<size_t>(slots);
}

int moe_place_experts(const moe_place_dims* pd, const int32_t* cap, const int64_t* A,
                      const int64_t* B, const double* D, const double* M, const int32_t* x0,
                      int32_t* x, int32_t* rank_experts, double* cost, void* stream) {
  if (pd == nullptr || cap == nullptr) return MOE_ERR_NULL;
  if (pd->L < 0 || pd->S < 1 || pd->E < 1 || pd->G < 1) return MOE_ERR_DIMS;
  if (pd->E > moe::kPlaceMaxExperts || pd->G > moe::kPlaceMaxRanks ||
      static_cast<int64_t>(pd->S) * pd->G > moe::kPlaceMaxSourceRanks ||
      moe::place_lds_bytes(pd->S, pd->E, pd->G) > static_cast<size_t>(moe::kPlaceMaxLdsBytes))
    return MOE_ERR_UNSUPPORTED;
  int64_t room = 0;
  for (int g = 0; g < pd->G; ++g) {
    if (cap[g] < 0) return MOE_ERR_DIMS;
    room += std::min(cap[g], pd->E);
  }
  if (room < pd->E) return MOE_ERR_DIMS;  // some expert would have no rank
  if (static_cast<int64_t>(pd->L) * pd->S * pd->E > (int64_t{1} << 40)) return MOE_ERR_UNSUPPORTED;
  if (pd->L == 0) return MOE_OK;
  if (!A || !D || !x0 || !x) return MOE_ERR_NULL;
  auto al = [](const void* p, uintptr_t n) { return (reinterpret_cast<uintptr_t>(p) & (n - 1)) == 0; };
  if (!al(A, 8) || !al(B, 8) || !al(D, 8) || !al(M, 8) || !al(cost, 8) || !al(x0, 4) || !al(x, 4) ||
      !al(rank_experts, 4))
    return MOE_ERR_ALIGN;
  moe::PlaceArgs a{};
  a.L = pd->L;
  a.S = pd->S;
  a.E = pd->E;
  a.G = pd->G;
  a.slots = static_cast<int>(moe_place_slots(pd, cap));
  a.alpha = pd->alpha;
  a.beta = pd->beta;
  a.gamma = pd->gamma;
  a.m_uniform = pd->m_uniform;
  a.cap = cap;
  a.A = A;
  a.B = B;
  a.D = D;
  a.M = M;
  a.x0 = x0;
  a.x = x;
  a.rank_experts = rank_experts;
  a.cost = cost;
  return status(moe::launch_place(a, static_cast<hipStream_t>(stream)));
}

int moe_window_stats(const moe_window_dims* wd, const int64_t* A, const int64_t* B, const int32_t* x,
                     const int32_t* home, const int32_t* engine, int64_t* remote, int64_t* total,
                     int64_t* rank_load, double* pressure, void* stream) {
  if (wd == nullptr) return MOE_ERR_NULL;
  if (wd->L < 0 || wd->S < 1 || wd->E < 1 || wd->G < 1 || wd->n_engines < 1) return MOE_ERR_DIMS;
  if (engine == nullptr && wd->n_engines != wd->G) return MOE_ERR_DIMS;
  if (wd->E > moe::kWindowMaxExperts || wd->G > moe::kWindowMaxRanks ||
      wd->n_engines > moe::kWindowMaxEngines ||
      static_cast<int64_t>(wd->L) * wd->S * wd->E > (int64_t{1} << 40))
    return MOE_ERR_UNSUPPORTED;
  if (wd->L > 0 && (!A || !x || !home || !remote || !total || !rank_load)) return MOE_ERR_NULL;
  auto al = [](const void* p, uintptr_t n) { return (reinterpret_cast<uintptr_t>(p) & (n - 1)) == 0; };
  if (!al(A, 8) || !al(B, 8) || !al(remote, 8) || !al(total, 8) || !al(rank_load, 8) || !al(pressure, 8) ||
      !al(x, 4) || !al(home, 4) || !al(engine, 4))
    return MOE_ERR_ALIGN;
  moe::WindowArgs a{wd->L, wd->S, wd->E, wd->G, wd->n_engines, A, B, x, home, engine,
                    remote, total, rank_load, pressure};
  return status(moe::launch_window(a, static_cast<hipStream_t>(stream)));
}

}  // extern "C"
