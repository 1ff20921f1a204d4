/*
 * moe.h -- C ABI of the MI355X (gfx950) MoE-layer hot path.
 *
 * One GPU's Mixture-of-Experts layer, the data-parallel path that source-aware
 * expert placement acts on: every token is tagged with the DP engine it
 * entered through, routed to its top-k experts, counted into the
 * source x expert matrix, dispatched to the experts hosted on this GPU, run
 * through their SwiGLU feed-forward networks and combined back into token
 * order.
 *
 * Conventions shared by every entry point
 *  - All array arguments are DEVICE pointers; moe_dims, moe_weights and
 *    moe_taps structs are HOST pointers read during the call only.
 *  - The caller owns every buffer.  The library never allocates, frees or
 *    synchronises; each call only enqueues kernels on `stream` (a hipStream_t
 *    passed as void*, NULL = the default stream) and returns.  Results are
 *    ready when the stream reaches them.
 *  - Process-wide state: per-device caches of fixed facts, each written
 *    once per device with atomic operations (so concurrent first calls are
 *    safe): a bit per device for every kernel whose LDS limit has been
 *    raised, the compute-unit count of each device, which sizes the expert
 *    GEMMs' persistent grids, and the address of each device's copy of
 *    moe_forward_noalloc's scratch array.  That array is the only mutable
 *    device state the library owns; only moe_forward_noalloc uses it.
 *  - Every check below is made on the host before anything is enqueued; a
 *    call that returns an error has enqueued nothing.  MOE_ERR_DEVICE means a
 *    launch failed after earlier launches of the same call may have been
 *    enqueued.
 *  - Data-dependent sizes (rows routed to each local expert) never leave the
 *    device: buffers indexed by routed rows are sized for the capacity T*k.
 *  - bf16 values are raw IEEE bf16 bit patterns (moe_bf16).  Every bf16 and
 *    fp32 array must be 16-byte aligned with rows whose byte length is a
 *    multiple of 16 (H and I multiples of 8), or the call returns
 *    MOE_ERR_ALIGN / MOE_ERR_UNSUPPORTED.
 *  - Calls are re-entrant.  Calls that overlap on different streams may share
 *    read-only inputs and the `counts` matrix (integer atomics); they must not
 *    share outputs or workspace.
 */
#ifndef MOE_H
#define MOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MOE_ABI_VERSION 2

typedef uint16_t moe_bf16;

/* Status codes returned by every entry point. */
enum moe_status {
    MOE_OK = 0,
    MOE_ERR_NULL = -1,        /* a required pointer is NULL */
    MOE_ERR_DIMS = -2,        /* inconsistent or negative dimensions */
    MOE_ERR_UNSUPPORTED = -3, /* valid, but beyond the kernels' limits */
    MOE_ERR_WORKSPACE = -4,   /* workspace missing or smaller than required */
    MOE_ERR_DEVICE = -5,      /* a kernel launch failed (e.g. not a gfx950 device) */
    MOE_ERR_ALIGN = -6        /* a pointer is not aligned as its entry point requires */
};

/*
 * Problem sizes (the paper's notation where it has one).
 *   T         tokens in the batch; each carries a source DP engine id (Sec. 1,
 *             Sec. 5.1: the "source" of the MoE traffic).
 *   H         hidden size.
 *   E         routed experts the router chooses among (gating width).
 *   k         experts selected per token (top-k, Sec. 2.1), 1 <= k <= E.
 *   I         intermediate size of a routed expert's SwiGLU FFN.
 *   S         number of source DP engines; source ids lie in [0, S).
 *   E_local   experts hosted on this GPU (its slice of the placement
 *             x_{l,e,g}, Sec. 5.2), 1 <= E_local <= E.
 *   n_shared  always-on shared experts applied to every token (0 = none).
 *   I_shared  intermediate size of each shared expert (ignored if n_shared=0).
 *   flags     the router's gate function, a moe_gate value (its parameters
 *             travel in moe_gating).
 * Kernel limits (MOE_ERR_UNSUPPORTED beyond them, decided on the host by
 * moe_validate and by every entry point before it enqueues anything):
 * E <= 1024, k <= 32, H, I, I_shared multiples of 8, T*k < 2^31, and the
 * 32-bit byte offsets of the expert GEMMs: within one expert's weight
 * matrices (about N*K*2 bytes), within a 256-row tile of activations or
 * outputs (257*max(H, I, n_shared*I_shared)*2 bytes), and, in moe_forward,
 * whose gate/up GEMM reads token rows through the dispatch list, within x
 * (T*H*2 < 2^31, i.e. T < 149,797 at H = 7168; moe_expert_ffn reads its
 * gathered rows tile by tile and has no such bound).
 */
typedef struct moe_dims {
    int32_t T, H, E, k, I, S, E_local, n_shared, I_shared, flags;
} moe_dims;

/*
 * Expert weights in nn.Linear layout (output features x input features),
 * bf16, row-major, stacked by LOCAL SLOT (slot s holds global expert
 * local_experts[s]):
 *   w_gate, w_up  [E_local][I][H]       w_down  [E_local][H][I]
 *   sh_gate, sh_up [n_shared][I_shared][H]   sh_down [n_shared][H][I_shared]
 * The shared pointers may be NULL when n_shared == 0.
 */
typedef struct moe_weights {
    const moe_bf16 *w_gate, *w_up, *w_down;
    const moe_bf16 *sh_gate, *sh_up, *sh_down;
} moe_weights;

/*
 * Gating variants (Sec. 2.1 requires a router that picks each token's top-k
 * experts; it does not fix the gating function, so three common ones are
 * offered).  moe_dims.flags selects one:
 *   MOE_GATE_SOFTMAX_TOPK  the softmax of the k selected logits, renormalised
 *                          over them (the default; selection on the logits);
 *   MOE_GATE_SOFTMAX       the softmax over all E logits evaluated at the k
 *                          selected experts, not renormalised (selection on
 *                          the logits);
 *   MOE_GATE_SIGMOID       sigmoid scores s_e = sigma(l_e), evaluated in fp64
 *                          and rounded to fp32; selection on s_e + bias_e
 *                          (fp32; the bias moves the selection only), gates
 *                          s_j / sum of the k selected s.
 * The moe_gating struct, nullable for no bias, scale 1 and no group limit, adds:
 *   bias          [E] fp32 device, nullable, MOE_GATE_SIGMOID only.
 *   routed_scale  every gate is multiplied by it.
 *   n_group, topk_group  group-limited selection when n_group > 1: the
 *                 experts form n_group groups of E / n_group consecutive ids;
 *                 a group's score is the fp32 sum of its two first selection
 *                 values in selection order (the single value when groups
 *                 hold one expert); only the topk_group first groups by
 *                 score (ties to the lower group) stay, and the k experts are
 *                 chosen among theirs.  Requires E % n_group == 0,
 *                 n_group <= 64, 1 <= topk_group <= n_group and
 *                 k <= topk_group * E / n_group.
 * Selection always orders by value descending, lower index first, NaN last.
 */
enum moe_gate { MOE_GATE_SOFTMAX_TOPK = 0, MOE_GATE_SOFTMAX = 1, MOE_GATE_SIGMOID = 2 };

typedef struct moe_gating {
    const float *bias;
    float routed_scale;
    int32_t n_group, topk_group;
} moe_gating;

/* Which entry point a workspace size refers to. */
enum moe_entry { MOE_ENTRY_PERMUTE = 1, MOE_ENTRY_EXPERT_FFN = 2, MOE_ENTRY_FORWARD = 3 };

/* Stages of moe_forward, for the optional timing events of moe_taps. */
enum moe_stage {
    MOE_STAGE_ROUTE = 0,    /* top-k gating (+ the source x expert counts when T*k <= 512) */
    MOE_STAGE_PERMUTE = 1,  /* slot counts (+ the source x expert counts when T*k > 512),
                               offsets, stable dispatch order */
    MOE_STAGE_FFN_UP = 2,   /* gate/up GEMM with the SwiGLU epilogue (routed, then shared) */
    MOE_STAGE_FFN_DOWN = 3, /* down GEMM (routed, then shared) */
    MOE_STAGE_COMBINE = 4,  /* weighted combine back to token order */
    MOE_NUM_STAGES = 5
};

/*
 * Optional extra outputs of moe_forward; every field may be NULL.
 *   topk_idx [T][k], topk_w [T][k], offsets [E_local+1], perm_token [T*k]
 *   (first offsets[E_local] entries valid), inv_pos [T*k]: copies of the
 *   intermediate results with the meaning given at the entry points below.
 *   expert_load [E]: set (=) to this call's per-expert load B.
 *   events[2*s], events[2*s+1]: hipEvent_t handles recorded on `stream`
 *   immediately before the first and after the last kernel of stage s.
 */
typedef struct moe_taps {
    int32_t *topk_idx;
    float *topk_w;
    int32_t *expert_load;
    int32_t *offsets;
    int32_t *perm_token;
    int32_t *inv_pos;
    void *events[2 * MOE_NUM_STAGES];
} moe_taps;

/* MOE_ABI_VERSION of the built library. */
int moe_abi_version(void);

/* Static text for a status code (never NULL). */
const char *moe_strerror(int status);

/*
 * Bytes of workspace `entry` needs for these sizes (0 when the dimensions are
 * invalid or beyond that entry point's limits; moe_validate says why).  Host only, no HIP call.  The workspace is
 * device memory owned by the caller, at least 256-byte aligned; its contents
 * need no initialisation and are undefined after the call.
 */
size_t moe_workspace_bytes(const moe_dims *dims, int entry);

/*
 * Host-only check of dims against the limits of entry point `entry` (0: of
 * every entry point) and, when entry != 0, of ws_bytes against
 * moe_workspace_bytes(dims, entry).  Returns MOE_OK or the status the entry
 * point would return for these sizes.  Makes no HIP call.
 */
int moe_validate(const moe_dims *dims, int entry, size_t ws_bytes);

/*
 * Top-k gating (Sec. 2.1: the router selects the top-k experts of each token).
 *   gating    nullable host struct: the parameters of the gate function that
 *             dims->flags selects (see moe_gating).
 *   logits    [T][E] fp32, row-major.
 *   topk_idx  [T][k] int32 out: the k selected experts of each token, ordered
 *             by selection value descending; equal values (-0.0 equals +0.0)
 *             go to the lower expert index; NaN ranks below every number.
 *   topk_w    [T][k] fp32 out: the gates (with the default gate function:
 *             the softmax of the selected logits renormalised over the k
 *             selected, NaN when the largest selected logit is not finite).
 * Uses T, E, k, flags.  T = 0 is a no-op.
 */
int moe_route(const moe_dims *dims, const moe_gating *gating,
              const float *logits, int32_t *topk_idx, float *topk_w,
              void *stream);

/*
 * Source-aware routing statistics (Sec. 5.1: the source x expert matrix
 * A_{l,s,e} and the aggregate load B_{l,e}).
 *   src          [T] int32: source DP engine of each token, expected in [0, S).
 *   topk_idx     [T][k] int32: expert ids, expected in [0, E).
 *   counts       [S][E] int64, ACCUMULATED (+=): one per pair (t, j) with
 *                src[t] = s and topk_idx[t][j] = e.  The caller keeps one
 *                buffer per layer and zeroes it to start a profiling window.
 *   expert_load  [E] int32, nullable, SET (=) to this call's column sums of
 *                the added counts.
 * A pair whose source or expert id is out of range is not counted (the call
 * stays in bounds; it does not report the bad id).  Uses T, E, k, S.
 */
int moe_route_stats(const moe_dims *dims, const int32_t *src,
                    const int32_t *topk_idx, int64_t *counts,
                    int32_t *expert_load, void *stream);

/*
 * Dispatch to the local experts (Sec. 2.1 dispatch; Sec. 5.2 placement slice).
 *   local_experts [E_local] int32, nullable: global expert hosted in each local
 *                 slot, distinct and in [0, E).  NULL means slot = expert id
 *                 and requires E_local == E.
 *   offsets       [E_local+1] int32 out: slot s owns rows
 *                 [offsets[s], offsets[s+1]); offsets[E_local] = R, the number
 *                 of pairs routed to local experts.
 *   perm_token    [T*k] int32 out: row r < R holds token perm_token[r]; rows
 *                 follow slot order, tokens ascending within a slot.
 *   inv_pos       [T*k] int32 out: row of pair (t, j) at t*k+j, or -1 when its
 *                 expert is not hosted here.
 *   x             [T][H] bf16 and x_perm [T*k][H] bf16 out: x_perm[r] =
 *                 x[perm_token[r]]; both may be NULL to skip the row gather.
 *   ws            MOE_ENTRY_PERMUTE workspace.
 * Expert ids outside [0, E) are treated as remote.  T = 0 sets offsets to 0.
 */
int moe_permute(const moe_dims *dims, const int32_t *topk_idx,
                const int32_t *local_experts, const moe_bf16 *x,
                int32_t *offsets, int32_t *perm_token, int32_t *inv_pos,
                moe_bf16 *x_perm, void *ws, size_t ws_bytes, void *stream);

/*
 * The experts' SwiGLU feed-forward networks as grouped GEMMs (Sec. 2.1: each
 * token activates only its experts' feed-forward parameters):
 *   y_perm[r] = W_down[s] (silu(W_gate[s] x_perm[r]) * (W_up[s] x_perm[r]))
 * for every row r in [offsets[s], offsets[s+1]), silu(z) = z / (1 + e^-z),
 * with fp32 accumulation and the intermediate rounded to bf16, and
 *   y_shared[t] = sum_q FFN^shared_q(x[t])   (fp32 sum, then bf16)
 * when n_shared > 0.
 *   x_perm   [T*k][H] bf16, rows [0, offsets[E_local]) read.
 *   offsets  [E_local+1] int32 as written by moe_permute.
 *   weights  see moe_weights.
 *   x        [T][H] bf16 (read only when n_shared > 0).
 *   y_perm   [T*k][H] bf16 out, rows [0, offsets[E_local]) written.
 *   y_shared [T][H] bf16 out (required when n_shared > 0, else ignored).
 *   ws       MOE_ENTRY_EXPERT_FFN workspace.
 */
int moe_expert_ffn(const moe_dims *dims, const moe_bf16 *x_perm,
                   const int32_t *offsets, const moe_weights *weights,
                   const moe_bf16 *x, moe_bf16 *y_perm, moe_bf16 *y_shared,
                   void *ws, size_t ws_bytes, void *stream);

/*
 * Weighted combine back to token order (Sec. 2.1: expert outputs are
 * combined and returned):
 *   out[t] = sum_{j<k, inv_pos[t*k+j] >= 0} topk_w[t][j] * y_perm[inv_pos[t*k+j]]
 *            + y_shared[t]
 * accumulated in fp32 in j order, then rounded to bf16.  Tokens none of whose
 * experts are local get y_shared[t] (or zeros).
 *   y_perm [T*k][H] bf16; inv_pos [T*k] int32 (entries must be -1 or a row
 *   written by moe_expert_ffn); topk_w [T][k] fp32; y_shared [T][H] bf16,
 *   nullable; out [T][H] bf16 out.
 */
int moe_combine(const moe_dims *dims, const moe_bf16 *y_perm,
                const int32_t *inv_pos, const float *topk_w,
                const moe_bf16 *y_shared, moe_bf16 *out, void *stream);

/*
 * The whole layer: moe_route (+ moe_route_stats) -> moe_permute ->
 * moe_expert_ffn -> moe_combine, with the intermediates in the workspace.
 *   gating as in moe_route;
 *   logits [T][E] fp32; src [T] int32 (nullable when counts is NULL);
 *   x [T][H] bf16; local_experts as in moe_permute; weights as in
 *   moe_expert_ffn;
 *   counts [S][E] int64, nullable: accumulated as in moe_route_stats (NULL
 *          skips the statistics);
 *   out [T][H] bf16 out: the layer output for this GPU's experts
 *          (plus the shared experts);
 *   taps   nullable host struct of optional extra outputs and events;
 *   ws     MOE_ENTRY_FORWARD workspace.
 */
int moe_forward(const moe_dims *dims, const moe_gating *gating,
                const float *logits, const int32_t *src,
                const moe_bf16 *x, const int32_t *local_experts,
                const moe_weights *weights, int64_t *counts, moe_bf16 *out,
                const moe_taps *taps, void *ws, size_t ws_bytes, void *stream);

/*
 * moe_forward without a caller workspace, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, hosts
 * that forbid allocation): the forward workspace lives in a library-owned
 * device array of MOE_NOALLOC_SCRATCH_BYTES (32 MiB), one copy per device,
 * held by every device the library runs on until the process ends.  The
 * call allocates and frees nothing; the caller still passes every input and
 * output.  Arguments and results are those of moe_forward.
 *   - Sizes whose forward workspace (moe_workspace_bytes(dims,
 *     MOE_ENTRY_FORWARD)) exceeds MOE_NOALLOC_SCRATCH_BYTES return
 *     MOE_ERR_WORKSPACE before anything is enqueued: decode-sized batches
 *     fit (64 tokens of a hidden-4096, intermediate-14336, top-2 layer need
 *     about 12 MB).
 *   - `stream` must belong to the current device (else MOE_ERR_DEVICE); the
 *     current device's copy of the array is used.
 *   - Every call on a device shares that device's array, which keeps the
 *     last call's contents: calls that overlap on one device, on any
 *     streams, race and must be serialised by the caller.
 */
#define MOE_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)

int moe_forward_noalloc(const moe_dims *dims, const moe_gating *gating,
                        const float *logits, const int32_t *src,
                        const moe_bf16 *x, const int32_t *local_experts,
                        const moe_weights *weights, int64_t *counts,
                        moe_bf16 *out, const moe_taps *taps, void *stream);

/*
 * ---- Source-aware expert placement (Sec. 5.2 objective, Sec. 5.3 greedy) ---
 *
 * At the end of a profiling window the placement manager turns the window's
 * statistics into a new expert placement for every layer.  The objective it
 * trades off (Sec. 5.2), for one layer with placement x_{e,g} in {0, 1}:
 *   L_g    = sum_e B_e x_{e,g},  Lbar = (1/G) sum_g L_g
 *   C_load = sum_g (L_g - Lbar)^2
 *   C_comm = sum_s sum_e sum_g A_{s,e} D_{s,g} x_{e,g}
 *   C_mig  = sum_e sum_g M_{e,g} |x_{e,g} - x^0_{e,g}|
 * The online heuristic (Sec. 5.3) visits the experts hottest first (aggregate
 * load B descending, then source-aware volume sum_s A descending, then lower
 * expert index) and gives each one the rank with spare capacity whose score
 *   S_{e,g} = alpha C^comm_{e,g} + beta C^load_{e,g} + gamma C^mig_{e,g}
 * is lowest, where each term is the amount by which the matching objective
 * term grows when e joins g, given the experts placed before it:
 *   C^comm_{e,g} = sum_s A_{s,e} D_{s,g}                 (summed in s order)
 *   C^load_{e,g} = (L_g + B_e - Lbar)^2 - (L_g - Lbar)^2 (L_g: load placed on g
 *                  so far; Lbar = (sum_e B_e) / G, the final average)
 *   C^mig_{e,g}  = 0 when g = x^0_e, else M_{e,g} + M_{e,x^0_e} (the second
 *                  term only when x^0_e is a rank)
 * Equal scores go to the expert's current rank, then to the rank with fewer
 * experts placed so far, then to the lower rank index.  Scores are fp64,
 * evaluated exactly in the order written (alpha C^comm, + beta C^load,
 * + gamma C^mig) without fused multiply-adds; a NaN score counts as +inf.
 * The paper calibrates (alpha, beta, gamma) = (1.0, 0.0025, 1.0) (Sec. 6).
 */
typedef struct moe_place_dims {
    int32_t L;    /* layers placed by one call, >= 0 */
    int32_t S;    /* source DP engines, >= 1 */
    int32_t E;    /* experts per layer, 1..1024 */
    int32_t G;    /* EP ranks, 1..64 */
    double alpha, beta, gamma;  /* score weights */
    double m_uniform;           /* M_{e,g} everywhere when M is NULL */
} moe_place_dims;

/*
 * Row length of moe_place_experts' rank_experts output: the largest number of
 * experts one rank can hold, max_g min(cap[g], E) (0 for NULL arguments or
 * E, G < 1).  Host only, no HIP call.
 */
size_t moe_place_slots(const moe_place_dims *dims, const int32_t *cap);

/*
 * New expert placement for L layers, one workgroup per layer.
 *   cap           [G] int32 HOST array: experts rank g can host per layer,
 *                 >= 0, with sum_g min(cap[g], E) >= E (else MOE_ERR_DIMS).
 *   A             [L][S][E] int64: the window's source x expert counts (the
 *                 per-layer `counts` of moe_route_stats, stacked).
 *   B             [L][E] int64, nullable: aggregate loads; NULL = the column
 *                 sums of A.
 *   D             [S][G] fp64: communication cost from source s to rank g.
 *   M             [L][E][G] fp64, nullable: cost of moving expert e to rank
 *                 g; NULL = dims->m_uniform everywhere.
 *   x0            [L][E] int32: rank hosting each expert now; a value outside
 *                 [0, G) means the expert is hosted nowhere yet.
 *   x             [L][E] int32 out: the new rank of each expert.
 *   rank_experts  [L][G][slots] int32 out, nullable: the experts of each rank
 *                 in ascending id order, padded with -1 (slots =
 *                 moe_place_slots); the first entries of a row are the
 *                 local_experts list moe_forward takes on that rank.
 *   cost          [L][3] fp64 out, nullable: C_comm, C_load, C_mig of the new
 *                 placement (sums in an unspecified order).
 * Limits (MOE_ERR_UNSUPPORTED beyond them): E <= 1024, G <= 64, S*G <= 4096.
 * int64 and fp64 arrays must be 8-byte aligned, int32 arrays 4-byte aligned
 * (MOE_ERR_ALIGN).  Counts are converted to fp64 for the scores (exact below
 * 2^53).  L = 0 is a no-op.
 */
int moe_place_experts(const moe_place_dims *dims, const int32_t *cap,
                      const int64_t *A, const int64_t *B, const double *D,
                      const double *M, const int32_t *x0, int32_t *x,
                      int32_t *rank_experts, double *cost, void *stream);

/*
 * ---- Window diagnostics under a placement (Sec. 2.2 Fig. 4; Sec. 4.1; Sec. 6)
 *
 * What a profiling window's statistics say about a placement x (for instance
 * the current one, or the one moe_place_experts proposes):
 *   - the traffic of each source that crosses to experts outside the source's
 *     own rank (the share of a DP group's MoE traffic sent to remote DP groups
 *     that motivates source-aware placement, Sec. 2.2, Fig. 4);
 *   - the token load each rank's experts process;
 *   - the MoE pressure each DP engine reports to the scheduler (Sec. 4.1): the
 *     token-equivalent expert load of the engine's ranks, all layers of the
 *     window, divided by the average over engines (1.0 = average; Sec. 6
 *     feeds it back as a relative penalty).
 */
typedef struct moe_window_dims {
    int32_t L;          /* layers, >= 0 */
    int32_t S;          /* source DP engines, >= 1 */
    int32_t E;          /* experts per layer, 1..8192 */
    int32_t G;          /* EP ranks, 1..1024 */
    int32_t n_engines;  /* DP engines the ranks belong to, 1..1024 */
} moe_window_dims;

/*
 *   A          [L][S][E] int64: the window's source x expert counts.
 *   B          [L][E] int64, nullable: aggregate loads (NULL = column sums of A).
 *   x          [L][E] int32: the rank hosting each expert; a value outside
 *              [0, G) hosts it nowhere (its tokens are remote for every
 *              source and load no rank).
 *   home       [S] int32: the EP rank co-located with each source's DP engine;
 *              outside [0, G) makes all of that source's traffic remote.
 *   engine     [G] int32, nullable: the DP engine (TP group) each rank belongs
 *              to, ranks mapped outside [0, n_engines) belong to none; NULL
 *              means rank g is engine g and requires n_engines == G.
 *   remote     [L][S] int64 out: sum_e A[l][s][e] over experts not on home[s].
 *   total      [L][S] int64 out: sum_e A[l][s][e].
 *   rank_load  [L][G] int64 out: sum of B[l][e] over the experts on rank g.
 *   pressure   [n_engines] fp64 out, nullable: engine load (its ranks'
 *              rank_load over all layers) / (all engines' load / n_engines),
 *              one IEEE division each; 0 when there is no load at all.
 * Integer results are exact (sums of int64, any order).  int64 and fp64
 * arrays 8-byte aligned, int32 arrays 4-byte aligned (MOE_ERR_ALIGN).  With
 * L = 0 only the pressure (all zeros) is written.
 */
int moe_window_stats(const moe_window_dims *dims, const int64_t *A,
                     const int64_t *B, const int32_t *x, const int32_t *home,
                     const int32_t *engine, int64_t *remote, int64_t *total,
                     int64_t *rank_load, double *pressure, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* MOE_H */
