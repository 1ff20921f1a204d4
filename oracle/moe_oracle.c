/*
 * moe_oracle.c -- plain CPU oracle for one GPU's MoE layer.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may call, link or
 * load this file; only the tests, the smoke check and the benchmark's CPU
 * baseline use it.  It shares no code, header, table or constant with the HIP
 * library: it is written straight from the definitions, single-threaded, with
 * no blocking, fusion or reordering, and accumulates in fp64.
 *
 * What the layer computes (the paper names the steps but never writes their
 * arithmetic; the readings taken where it is silent are listed with the
 * design notes):
 *   - a router picks the top-k experts of each token (Sec. 2.1);
 *   - each token carries the DP engine ("source") it entered through, and the
 *     layer counts A[s][e] = tokens from source s routed to expert e, plus the
 *     aggregate load B[e] = tokens routed to expert e (Sec. 5.1, the matrices
 *     A_{l,s,e} and B_{l,e});
 *   - tokens are dispatched to the experts hosted on this GPU, i.e. the slice
 *     of the placement x_{l,e,g} that belongs to it (Sec. 5.2), run through
 *     those experts' feed-forward networks and combined back (Sec. 2.1).
 *
 * Every public function returns 0 on success and a negative code on a bad
 * argument or input (-2: dimensions, -6: data outside its documented range).
 * Parity status of each function is stated at the function.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_OK 0
#define ORACLE_ERR_DIMS (-2)
#define ORACLE_ERR_DATA (-6)
#define ORACLE_ERR_NOMEM (-7)

/* A bf16 value is the top half of an fp32 word: widening is exact. */
static double bf16_value(uint16_t bits)
{
    uint32_t u = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/*
 * The order in which experts are selected (Sec. 2.1, "top-k experts for each
 * token"; the paper does not say how equal logits are resolved).  Expert a
 * comes before expert b when its logit is larger; equal logits (-0.0 equals
 * +0.0 under IEEE comparison) go to the lower index, the same lexicographic
 * lower-index rule the paper uses for its own tie-breaks (Alg. 1).  A NaN
 * logit comes after every number, NaNs among themselves by index.
 */
static int comes_before(float a, int ia, float b, int ib)
{
    int a_nan = isnan(a), b_nan = isnan(b);
    if (a_nan || b_nan) {
        if (a_nan && b_nan)
            return ia < ib;
        return b_nan;
    }
    if (a != b)
        return a > b;
    return ia < ib;
}

/*
 * Top-k routing (Sec. 2.1).  For each token t, topk_idx[t][0..k-1] are the
 * first k experts of the order above, in that order.  The gate of the j-th
 * selected expert is the softmax of the selected logits renormalised over the
 * k of them: w_j = exp(l_j - m) / sum_j' exp(l_j' - m) with m the largest
 * selected logit.  Gates are defined when the selected logits are finite or
 * -inf with a finite maximum; otherwise they come out NaN.
 *
 * Pinned by: brute-force subset enumeration on tiny rows, numpy's stable
 * argsort and argmax, hand-derived tie / signed-zero / NaN / -inf rows, and
 * closed-form gates (k = 1, k = 2 logistic form, sum to one).
 */
int oracle_route(int T, int E, int k, const float *logits,
                 int32_t *topk_idx, double *topk_w)
{
    if (T < 0 || E < 1 || k < 1 || k > E)
        return ORACLE_ERR_DIMS;
    char *taken = (char *)malloc((size_t)E);
    if (!taken)
        return ORACLE_ERR_NOMEM;
    for (int t = 0; t < T; ++t) {
        const float *row = logits + (size_t)t * E;
        int32_t *idx = topk_idx + (size_t)t * k;
        memset(taken, 0, (size_t)E);
        /* selection: repeatedly take the first not-yet-taken expert */
        for (int j = 0; j < k; ++j) {
            int best = -1;
            for (int e = 0; e < E; ++e) {
                if (taken[e])
                    continue;
                if (best < 0 || comes_before(row[e], e, row[best], best))
                    best = e;
            }
            taken[best] = 1;
            idx[j] = best;
        }
        /* gates: softmax over the k selected logits */
        double m = (double)row[idx[0]];
        double sum = 0.0;
        for (int j = 0; j < k; ++j)
            sum += exp((double)row[idx[j]] - m);
        for (int j = 0; j < k; ++j)
            topk_w[(size_t)t * k + j] = exp((double)row[idx[j]] - m) / sum;
    }
    free(taken);
    return ORACLE_OK;
}

/*
 * Gating variants (Sec. 2.1 names a router that picks each token's top-k
 * experts but not its gating function; three common ones are written out
 * here).  gate selects:
 *   0  softmax over the k selected logits (renormalised; oracle_route);
 *   1  softmax over all E logits, evaluated at the k selected experts (not
 *      renormalised): w_j = exp(l_j - M) / sum_e exp(l_e - M), M the largest
 *      logit that is a number;
 *   2  sigmoid scores s_e = sigma(l_e), evaluated in fp64 and rounded to fp32;
 *      experts are selected by s_e + bias_e (fp32 sum; bias nullable, used
 *      for the selection only) and weighted w_j = s_j / sum_j' s_j'.
 * Selection is by the selection value c_e (l_e for gates 0 and 1, s_e + bias_e
 * for gate 2) under the total order of comes_before (value descending, lower
 * index first, NaN last).  With n_group > 1 the experts form n_group groups
 * of E / n_group consecutive ids; a group's score is the fp32 sum of its two
 * first selection values in that order (its one value when groups hold a
 * single expert); the first topk_group groups in the order of comes_before
 * over group scores stay, and the k experts are selected among theirs.  All
 * gates are finally multiplied by scale.
 *
 * Pinned by: brute-force enumeration of the kept group set and of the
 * selected experts; the full softmax of a library routine evaluated at the
 * selected experts; sigmoid gates in closed form; the bias moving the
 * selection but not the gates; n_group = 1 and topk_group = n_group reducing
 * to the ungrouped selection; a hand-worked grouped example.
 */
int oracle_route_gated(int T, int E, int k, int gate, const float *logits,
                       const float *bias, double scale, int n_group,
                       int topk_group, int32_t *topk_idx, double *topk_w)
{
    if (T < 0 || E < 1 || k < 1 || k > E || gate < 0 || gate > 2)
        return ORACLE_ERR_DIMS;
    if (bias && gate != 2)
        return ORACLE_ERR_DIMS;
    int grouped = n_group > 1;
    int gsz = grouped ? E / n_group : E;
    if (grouped && (E % n_group != 0 || topk_group < 1 || topk_group > n_group ||
                    k > topk_group * gsz))
        return ORACLE_ERR_DIMS;
    int rc = ORACLE_OK;
    float *c = (float *)malloc(sizeof(float) * (size_t)E);
    double *sg = (double *)malloc(sizeof(double) * (size_t)E);
    char *allowed = (char *)malloc((size_t)E);
    char *taken = (char *)malloc((size_t)E);
    float *gscore = (float *)malloc(sizeof(float) * (size_t)(grouped ? n_group : 1));
    char *gtaken = (char *)malloc((size_t)(grouped ? n_group : 1));
    if (!c || !sg || !allowed || !taken || !gscore || !gtaken) {
        rc = ORACLE_ERR_NOMEM;
        goto done;
    }
    for (int t = 0; t < T; ++t) {
        const float *row = logits + (size_t)t * E;
        int32_t *idx = topk_idx + (size_t)t * k;
        double *w = topk_w + (size_t)t * k;
        /* selection values */
        for (int e = 0; e < E; ++e) {
            if (gate == 2) {
                float s = (float)(1.0 / (1.0 + exp(-(double)row[e])));
                sg[e] = (double)s;
                c[e] = bias ? s + bias[e] : s;
            } else {
                c[e] = row[e];
            }
            allowed[e] = 1;
        }
        /* group limit: keep the topk_group best groups */
        if (grouped) {
            for (int q = 0; q < n_group; ++q) {
                int first = -1, second = -1;
                for (int e = q * gsz; e < (q + 1) * gsz; ++e) {
                    if (first < 0 || comes_before(c[e], e, c[first], first)) {
                        second = first;
                        first = e;
                    } else if (second < 0 || comes_before(c[e], e, c[second], second)) {
                        second = e;
                    }
                }
                gscore[q] = second < 0 ? c[first] : c[first] + c[second];
                gtaken[q] = 0;
            }
            for (int j = 0; j < topk_group; ++j) {
                int best = -1;
                for (int q = 0; q < n_group; ++q) {
                    if (gtaken[q])
                        continue;
                    if (best < 0 || comes_before(gscore[q], q, gscore[best], best))
                        best = q;
                }
                gtaken[best] = 1;
            }
            for (int e = 0; e < E; ++e)
                allowed[e] = gtaken[e / gsz];
        }
        /* the k first allowed experts */
        memset(taken, 0, (size_t)E);
        for (int j = 0; j < k; ++j) {
            int best = -1;
            for (int e = 0; e < E; ++e) {
                if (taken[e] || !allowed[e])
                    continue;
                if (best < 0 || comes_before(c[e], e, c[best], best))
                    best = e;
            }
            taken[best] = 1;
            idx[j] = best;
        }
        /* gates */
        if (gate == 0) {
            double m = (double)row[idx[0]];
            double sum = 0.0;
            for (int j = 0; j < k; ++j)
                sum += exp((double)row[idx[j]] - m);
            for (int j = 0; j < k; ++j)
                w[j] = exp((double)row[idx[j]] - m) / sum;
        } else if (gate == 1) {
            double m = NAN;
            for (int e = 0; e < E; ++e)
                if (!isnan(row[e]) && (isnan(m) || (double)row[e] > m))
                    m = (double)row[e];
            double sum = 0.0;
            for (int e = 0; e < E; ++e)
                sum += exp((double)row[e] - m);
            for (int j = 0; j < k; ++j)
                w[j] = exp((double)row[idx[j]] - m) / sum;
        } else {
            double sum = 0.0;
            for (int j = 0; j < k; ++j)
                sum += sg[idx[j]];
            for (int j = 0; j < k; ++j)
                w[j] = sg[idx[j]] / sum;
        }
        for (int j = 0; j < k; ++j)
            w[j] *= scale;
    }
done:
    free(c);
    free(sg);
    free(allowed);
    free(taken);
    free(gscore);
    free(gtaken);
    return rc;
}

/*
 * Source-aware routing statistics (Sec. 5.1).  counts is the S x E matrix A
 * of this layer and is accumulated (+=) so that successive calls form a
 * profiling window; counts[s][e] gains one for every selected pair (t, j)
 * with src[t] = s and topk_idx[t][j] = e.  expert_load (nullable) is set (=)
 * to this call's aggregate load B[e] = number of selected pairs with expert e.
 * Every source id must lie in [0, S) and every expert id in [0, E).
 *
 * Pinned by: hand-derived counts, total = T*k, row sums = k * tokens of the
 * source, column sums = numpy bincount of the expert ids.
 */
int oracle_route_stats(int T, int k, int S, int E, const int32_t *src,
                       const int32_t *topk_idx, int64_t *counts,
                       int32_t *expert_load)
{
    if (T < 0 || k < 1 || S < 1 || E < 1 || k > E)
        return ORACLE_ERR_DIMS;
    for (int t = 0; t < T; ++t) {
        if (src[t] < 0 || src[t] >= S)
            return ORACLE_ERR_DATA;
        for (int j = 0; j < k; ++j) {
            int32_t e = topk_idx[(size_t)t * k + j];
            if (e < 0 || e >= E)
                return ORACLE_ERR_DATA;
        }
    }
    if (expert_load)
        for (int e = 0; e < E; ++e)
            expert_load[e] = 0;
    for (int t = 0; t < T; ++t) {
        for (int j = 0; j < k; ++j) {
            int32_t e = topk_idx[(size_t)t * k + j];
            counts[(size_t)src[t] * E + e] += 1;
            if (expert_load)
                expert_load[e] += 1;
        }
    }
    return ORACLE_OK;
}

/*
 * Dispatch to the locally hosted experts (Secs. 2.1, 5.2).  This GPU hosts
 * the experts local_experts[0..E_local-1]; expert local_experts[s] occupies
 * local slot s (NULL means every expert, slot = expert id, E_local = E).  The
 * selected pairs whose expert is hosted here are sorted by slot with a stable
 * counting sort over (t, j) in token-major order:
 *   offsets[s]       first row of slot s, offsets[E_local] = R rows in total;
 *   perm_token[r]    the token whose hidden state goes to row r (r < R);
 *   inv_pos[t*k+j]   the row of pair (t, j), or -1 if its expert is remote.
 *
 * Pinned by: a hand-derived placement example, the bijection between local
 * pairs and rows, and numpy's stable argsort of the slot keys.
 */
int oracle_permute(int T, int k, int E, int E_local,
                   const int32_t *local_experts, const int32_t *topk_idx,
                   int32_t *offsets, int32_t *perm_token, int32_t *inv_pos)
{
    if (T < 0 || k < 1 || E < 1 || E_local < 1 || E_local > E || k > E)
        return ORACLE_ERR_DIMS;
    if (!local_experts && E_local != E)
        return ORACLE_ERR_DIMS;
    int32_t *slot_of = (int32_t *)malloc(sizeof(int32_t) * (size_t)E);
    int64_t *fill = (int64_t *)calloc((size_t)E_local, sizeof(int64_t));
    if (!slot_of || !fill) {
        free(slot_of);
        free(fill);
        return ORACLE_ERR_NOMEM;
    }
    int rc = ORACLE_OK;
    for (int e = 0; e < E; ++e)
        slot_of[e] = local_experts ? -1 : e;
    if (local_experts) {
        for (int s = 0; s < E_local; ++s) {
            int32_t e = local_experts[s];
            if (e < 0 || e >= E || slot_of[e] != -1) {
                rc = ORACLE_ERR_DATA;   /* out of range or hosted twice */
                goto done;
            }
            slot_of[e] = s;
        }
    }
    for (size_t p = 0; p < (size_t)T * k; ++p) {
        if (topk_idx[p] < 0 || topk_idx[p] >= E) {
            rc = ORACLE_ERR_DATA;
            goto done;
        }
    }
    /* count per slot, then exclusive prefix sum */
    for (size_t p = 0; p < (size_t)T * k; ++p) {
        int32_t s = slot_of[topk_idx[p]];
        if (s >= 0)
            fill[s] += 1;
    }
    offsets[0] = 0;
    for (int s = 0; s < E_local; ++s)
        offsets[s + 1] = offsets[s] + (int32_t)fill[s];
    /* place the pairs, visiting them in token-major order */
    memset(fill, 0, sizeof(int64_t) * (size_t)E_local);
    for (int t = 0; t < T; ++t) {
        for (int j = 0; j < k; ++j) {
            size_t p = (size_t)t * k + j;
            int32_t s = slot_of[topk_idx[p]];
            if (s < 0) {
                inv_pos[p] = -1;
                continue;
            }
            int32_t r = offsets[s] + (int32_t)fill[s];
            fill[s] += 1;
            perm_token[r] = t;
            inv_pos[p] = r;
        }
    }
done:
    free(slot_of);
    free(fill);
    return rc;
}

/* Row gather x_perm[r] = x[perm_token[r]] for r < R (bf16 bits copied). */
int oracle_gather_rows(int R, int H, const int32_t *perm_token,
                       const uint16_t *x, uint16_t *x_perm)
{
    if (R < 0 || H < 1)
        return ORACLE_ERR_DIMS;
    for (int r = 0; r < R; ++r)
        memcpy(x_perm + (size_t)r * H, x + (size_t)perm_token[r] * H,
               sizeof(uint16_t) * (size_t)H);
    return ORACLE_OK;
}

static double silu(double z)
{
    return z / (1.0 + exp(-z));
}

/*
 * First half of one expert's feed-forward network (the "feedforward
 * parameters" an expert holds, Sec. 2.1; the SwiGLU form is the workload's):
 *   h[i] = silu(g_i) * u_i,  g = W_gate x,  u = W_up x,  silu(z) = z/(1+e^-z)
 * with W_gate, W_up of shape [I][H] (row i holds the weights of output i).
 *
 * Pinned by: hand-derived saturated and silu(1) examples, linearity in W_up,
 * and the gate/up asymmetry.
 */
int oracle_swiglu_hidden(int H, int I, const uint16_t *x,
                         const uint16_t *w_gate, const uint16_t *w_up,
                         double *h)
{
    if (H < 1 || I < 1)
        return ORACLE_ERR_DIMS;
    for (int i = 0; i < I; ++i) {
        const uint16_t *wg = w_gate + (size_t)i * H;
        const uint16_t *wu = w_up + (size_t)i * H;
        double g = 0.0, u = 0.0;
        for (int c = 0; c < H; ++c) {
            double xc = bf16_value(x[c]);
            g += bf16_value(wg[c]) * xc;
            u += bf16_value(wu[c]) * xc;
        }
        h[i] = silu(g) * u;
    }
    return ORACLE_OK;
}

/* y = W v with W of shape [n_out][n_in] in bf16 and v, y in fp64. */
int oracle_linear(int n_out, int n_in, const uint16_t *w, const double *v,
                  double *y)
{
    if (n_out < 1 || n_in < 1)
        return ORACLE_ERR_DIMS;
    for (int o = 0; o < n_out; ++o) {
        const uint16_t *row = w + (size_t)o * n_in;
        double acc = 0.0;
        for (int c = 0; c < n_in; ++c)
            acc += bf16_value(row[c]) * v[c];
        y[o] = acc;
    }
    return ORACLE_OK;
}

/*
 * One expert's whole feed-forward network on one token:
 *   FFN(x) = W_down (silu(W_gate x) * (W_up x)),  W_down of shape [H][I].
 */
int oracle_swiglu_ffn(int H, int I, const uint16_t *x, const uint16_t *w_gate,
                      const uint16_t *w_up, const uint16_t *w_down, double *y)
{
    if (H < 1 || I < 1)
        return ORACLE_ERR_DIMS;
    double *h = (double *)malloc(sizeof(double) * (size_t)I);
    if (!h)
        return ORACLE_ERR_NOMEM;
    int rc = oracle_swiglu_hidden(H, I, x, w_gate, w_up, h);
    if (rc == ORACLE_OK)
        rc = oracle_linear(H, I, w_down, h, y);
    free(h);
    return rc;
}

/*
 * Expert outputs for a list of permuted rows: y[r] = FFN_{slot[r]}(x_rows[r]),
 * with the routed weights of the hosted slots stacked as [E_local][I][H]
 * (gate, up) and [E_local][H][I] (down).
 */
int oracle_ffn_rows(int n, int H, int I, int E_local, const int32_t *slot,
                    const uint16_t *x_rows, const uint16_t *w_gate,
                    const uint16_t *w_up, const uint16_t *w_down, double *y)
{
    if (n < 0 || H < 1 || I < 1 || E_local < 1)
        return ORACLE_ERR_DIMS;
    size_t wsz = (size_t)I * H;
    for (int r = 0; r < n; ++r) {
        if (slot[r] < 0 || slot[r] >= E_local)
            return ORACLE_ERR_DATA;
        int rc = oracle_swiglu_ffn(H, I, x_rows + (size_t)r * H,
                                   w_gate + (size_t)slot[r] * wsz,
                                   w_up + (size_t)slot[r] * wsz,
                                   w_down + (size_t)slot[r] * wsz,
                                   y + (size_t)r * H);
        if (rc != ORACLE_OK)
            return rc;
    }
    return ORACLE_OK;
}

/*
 * Combine back to token order (Sec. 2.1, outputs "combined and returned"):
 *   out[t] = sum_{j<k, inv_pos[t*k+j] >= 0} w[t][j] * y_perm[inv_pos[t*k+j]]
 *            + y_shared[t]                       (when y_shared is given)
 * y_perm and y_shared are bf16 bits, weights fp32, out fp64; j ascending.
 */
int oracle_combine(int T, int k, int H, int R, const uint16_t *y_perm,
                   const int32_t *inv_pos, const float *topk_w,
                   const uint16_t *y_shared, double *out)
{
    if (T < 0 || k < 1 || H < 1 || R < 0)
        return ORACLE_ERR_DIMS;
    for (int t = 0; t < T; ++t) {
        double *o = out + (size_t)t * H;
        for (int c = 0; c < H; ++c)
            o[c] = 0.0;
        for (int j = 0; j < k; ++j) {
            int32_t r = inv_pos[(size_t)t * k + j];
            if (r < 0)
                continue;
            if (r >= R)
                return ORACLE_ERR_DATA;
            double w = (double)topk_w[(size_t)t * k + j];
            for (int c = 0; c < H; ++c)
                o[c] += w * bf16_value(y_perm[(size_t)r * H + c]);
        }
        if (y_shared)
            for (int c = 0; c < H; ++c)
                o[c] += bf16_value(y_shared[(size_t)t * H + c]);
    }
    return ORACLE_OK;
}

/*
 * The whole layer for a list of tokens, straight from the definition and
 * never through a permutation:
 *   out[t] = sum_{j<k, expert hosted here} w_tj * FFN_{e_tj}(x_t)
 *            + sum_{q<n_shared} FFN^shared_q(x_t)
 * where (e_tj, w_tj) are the token's routing choice and gates (oracle_route
 * on its logit row), the routed sum runs over j ascending and the shared sum
 * over q ascending.  Tokens whose experts are all remote receive only the
 * shared part (zero without shared experts).
 *
 * The routing is oracle_route_gated with gate = dims[9] and the gating
 * parameters given (gate 0 with no bias, scale 1 and no group limit is
 * oracle_route).
 *
 * dims = {T, H, E, k, I, S, E_local, n_shared, I_shared, gate}; routed weights are
 * stacked by local slot, shared ones as [n_shared][I_shared][H] (gate, up)
 * and [n_shared][H][I_shared] (down).
 *
 * Pinned by: one-hot gates reduce to a single dense FFN; identical experts
 * reduce to one dense FFN (gates sum to one); splitting the experts over two
 * placements adds up to the placement that hosts them all.
 */
int oracle_forward_tokens(const int32_t *dims, int n_tok, const int32_t *tokens,
                          const float *logits, const uint16_t *x,
                          const int32_t *local_experts, const uint16_t *w_gate,
                          const uint16_t *w_up, const uint16_t *w_down,
                          const uint16_t *sh_gate, const uint16_t *sh_up,
                          const uint16_t *sh_down, const float *gate_bias,
                          double gate_scale, int n_group, int topk_group,
                          double *out)
{
    int T = dims[0], H = dims[1], E = dims[2], k = dims[3], I = dims[4];
    int E_local = dims[6], n_sh = dims[7], I_sh = dims[8], gate = dims[9];
    if (T < 0 || H < 1 || E < 1 || k < 1 || k > E || I < 1 || E_local < 1 ||
        E_local > E || n_sh < 0 || (n_sh > 0 && I_sh < 1) || n_tok < 0)
        return ORACLE_ERR_DIMS;
    if (!local_experts && E_local != E)
        return ORACLE_ERR_DIMS;
    int rc = ORACLE_OK;
    int32_t *slot_of = (int32_t *)malloc(sizeof(int32_t) * (size_t)E);
    int32_t *idx = (int32_t *)malloc(sizeof(int32_t) * (size_t)k);
    double *w = (double *)malloc(sizeof(double) * (size_t)k);
    double *y = (double *)malloc(sizeof(double) * (size_t)H);
    if (!slot_of || !idx || !w || !y) {
        rc = ORACLE_ERR_NOMEM;
        goto done;
    }
    for (int e = 0; e < E; ++e)
        slot_of[e] = local_experts ? -1 : e;
    if (local_experts) {
        for (int s = 0; s < E_local; ++s) {
            int32_t e = local_experts[s];
            if (e < 0 || e >= E || slot_of[e] != -1) {
                rc = ORACLE_ERR_DATA;
                goto done;
            }
            slot_of[e] = s;
        }
    }
    size_t wsz = (size_t)I * H, shsz = (size_t)I_sh * H;
    for (int n = 0; n < n_tok; ++n) {
        int t = tokens[n];
        if (t < 0 || t >= T) {
            rc = ORACLE_ERR_DATA;
            goto done;
        }
        const uint16_t *xt = x + (size_t)t * H;
        double *o = out + (size_t)n * H;
        rc = oracle_route_gated(1, E, k, gate, logits + (size_t)t * E, gate_bias,
                                gate_scale, n_group, topk_group, idx, w);
        if (rc != ORACLE_OK)
            goto done;
        for (int c = 0; c < H; ++c)
            o[c] = 0.0;
        for (int j = 0; j < k; ++j) {
            int32_t s = slot_of[idx[j]];
            if (s < 0)
                continue;
            rc = oracle_swiglu_ffn(H, I, xt, w_gate + (size_t)s * wsz,
                                   w_up + (size_t)s * wsz,
                                   w_down + (size_t)s * wsz, y);
            if (rc != ORACLE_OK)
                goto done;
            for (int c = 0; c < H; ++c)
                o[c] += w[j] * y[c];
        }
        for (int q = 0; q < n_sh; ++q) {
            rc = oracle_swiglu_ffn(H, I_sh, xt, sh_gate + (size_t)q * shsz,
                                   sh_up + (size_t)q * shsz,
                                   sh_down + (size_t)q * shsz, y);
            if (rc != ORACLE_OK)
                goto done;
            for (int c = 0; c < H; ++c)
                o[c] += y[c];
        }
    }
done:
    free(slot_of);
    free(idx);
    free(w);
    free(y);
    return rc;
}
