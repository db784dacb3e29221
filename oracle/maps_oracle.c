/*
 * CPU oracle of the MAPS scheduler core.  TEST INFRASTRUCTURE ONLY: the tests,
 * the smoke check and the benchmark's CPU-baseline leg may load it; the product
 * path never does.  It shares no code, header or table with the GPU library.
 *
 * Plain, slow and direct: every quantity is computed from its definition in
 * the paper, in 64-bit integers, one decoding step at a time.
 *
 *   calibration  Sec. 3.2, Eqs. (2)-(4): one-sided nonconformity score, the
 *                conformal rank ceil((1-alpha)(n+1)), the calibrated bound;
 *                applied per length bucket of the prediction, on a fixed
 *                calibration set or on each request's sliding window of the
 *                most recent completions (Sec. 3.2, Sec. 4).
 *   occupancy    Sec. 3.3 and App. A, Eqs. (8) and (10): the KV footprint of a
 *                request grows one token per decoding step ("token by token",
 *                Sec. 3.3) until its bound runs out.
 *   placement    Algorithm 1 / App. C: feasible decoders, minimum-queue choice,
 *                maximum-capacity fallback, round-robin when no bound exists
 *                (Eq. (9)), with the static block test replaced by the
 *                projected peak of the decoder's occupancy plus the arrival.
 *   static rule  Sec. 3.3 and Algorithm 1 as printed: block counts of the
 *                runtime state, B_need <= B_eff, and with reservation each
 *                dispatch reserving its B_need before the next arrival.
 *   local order  Sec. 3.3, Eq. (7): argsort of the queue by the bound, with
 *                starvation promotion, and the App. A admission rule (10)
 *                applied to the reordered queue.
 *
 * Readings of points the paper leaves open:
 *   - alpha is an integer in parts per million; the rank is an exact integer
 *     ceiling.  A rank above the bucket size gives an infinite quantile, and
 *     the bound is then the cap u_max.  Bounds are capped at u_max.
 *   - a request is bucketed by its prediction: #{edges <= pred}.
 *   - a resident with prompt p, generated g and bound U holds p+g+t tokens at
 *     future step t while t <= R = max(U-g, 0); an arrival with bound U holds
 *     p+t while t <= U.  Step 0 is the present.
 *   - feasible means peak <= capacity; ties go to the lowest decoder index.
 *   - a negative prediction means "no prediction": the bound is -1, and a
 *     negative bound routes the arrival round-robin.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_Q_INF INT32_MAX
#define ORACLE_POLICY_MQ 0
#define ORACLE_POLICY_MC 1

static int64_t max64(int64_t a, int64_t b) { return a > b ? a : b; }
static int64_t min64(int64_t a, int64_t b) { return a < b ? a : b; }

/* ------------------------------------------------------------------------ */
/* Calibration (Sec. 3.2)                                                    */
/* ------------------------------------------------------------------------ */

/* Length bucket of a prediction: the number of edges not above it. */
int32_t oracle_bucket(int32_t pred, const int32_t* edges, int32_t nb)
{
    int32_t b = 0;
    for (int32_t j = 0; j < nb - 1; ++j)
        if (edges[j] <= pred) b += 1;
    return b;
}

/* Eq. (3): k = ceil((1 - alpha) * (n + 1)), alpha = alpha_ppm / 10^6. */
int64_t oracle_conformal_rank(int64_t n, int32_t alpha_ppm)
{
    int64_t num = (int64_t)(1000000 - alpha_ppm) * (n + 1);
    return (num + 999999) / 1000000;
}

static int cmp_i64(const void* a, const void* b)
{
    int64_t x = *(const int64_t*)a, y = *(const int64_t*)b;
    return (x > y) - (x < y);
}

/* Eqs. (2)-(3) per bucket: q[b] is the k-th smallest score of bucket b
 * (1-indexed, multiset), or ORACLE_Q_INF when k exceeds the bucket size. */
int oracle_calibrate(const int32_t* pred, const int32_t* truth, int64_t n,
                     const int32_t* edges, int32_t nb, int32_t alpha_ppm,
                     int32_t* q_out, int32_t* count_out)
{
    if (nb < 1 || alpha_ppm <= 0 || alpha_ppm >= 1000000 || n < 0) return -1;
    int64_t* count = (int64_t*)calloc((size_t)nb, sizeof(int64_t));
    int64_t* start = (int64_t*)calloc((size_t)nb + 1, sizeof(int64_t));
    int64_t* fill = (int64_t*)calloc((size_t)nb, sizeof(int64_t));
    int64_t* scores = (int64_t*)malloc((size_t)(n > 0 ? n : 1) * sizeof(int64_t));
    if (!count || !start || !fill || !scores) return -2;

    for (int64_t i = 0; i < n; ++i) count[oracle_bucket(pred[i], edges, nb)] += 1;
    for (int32_t b = 0; b < nb; ++b) start[b + 1] = start[b] + count[b];
    for (int64_t i = 0; i < n; ++i) {
        int32_t b = oracle_bucket(pred[i], edges, nb);
        /* Eq. (2): s = (L - L_hat)_+ */
        int64_t s = max64(0, (int64_t)truth[i] - (int64_t)pred[i]);
        scores[start[b] + fill[b]] = s;
        fill[b] += 1;
    }
    for (int32_t b = 0; b < nb; ++b) {
        int64_t nb_b = count[b];
        qsort(scores + start[b], (size_t)nb_b, sizeof(int64_t), cmp_i64);
        int64_t k = oracle_conformal_rank(nb_b, alpha_ppm);
        q_out[b] = (k <= nb_b) ? (int32_t)scores[start[b] + k - 1] : ORACLE_Q_INF;
        count_out[b] = (int32_t)nb_b;
    }
    free(count); free(start); free(fill); free(scores);
    return 0;
}

/* Eq. (4): U = L_hat + q of the prediction's bucket, capped at u_max; an
 * infinite quantile gives u_max and a missing prediction (< 0) gives -1. */
void oracle_apply_bounds(const int32_t* pred, int64_t m, const int32_t* edges, int32_t nb,
                         const int32_t* q, int32_t u_max, int32_t* U_out)
{
    for (int64_t i = 0; i < m; ++i) {
        if (pred[i] < 0) { U_out[i] = -1; continue; }
        int32_t qb = q[oracle_bucket(pred[i], edges, nb)];
        if (qb == ORACLE_Q_INF) U_out[i] = u_max;
        else U_out[i] = (int32_t)min64((int64_t)pred[i] + qb, u_max);
    }
}

/* ------------------------------------------------------------------------ */
/* Sliding-window calibration (Sec. 3.2: the calibration set holds the most  */
/* recent completed requests; Sec. 4: a window of the 500 most recent)       */
/* ------------------------------------------------------------------------ */

/* Bounds for m requests, each calibrated on its own set: the `window` most
 * recent completions of the request's bucket among the first seen[j] entries
 * of the completion log (oldest first), or all of them when the bucket has
 * fewer.  Eqs. (2)-(3) on that set give q_out[j]: the k-th smallest score,
 * k = ceil((1-alpha)(n_w+1)) for a set of n_w scores, ORACLE_Q_INF when k
 * exceeds n_w (an empty set included); a request without a prediction gets
 * q_out = -1 and U_out = -1.  U_out follows Eq. (4) as in oracle_apply_bounds.
 * Returns -1 on bad arguments, -2 when out of memory, -3 when a seen count
 * lies outside [0, n], -4 for a negative length in the log. */
int oracle_calibrate_window(const int32_t* pred, const int32_t* truth, int64_t n,
                            const int32_t* edges, int32_t nb, int32_t window, int32_t alpha_ppm,
                            const int32_t* apply_pred, const int64_t* seen, int64_t m,
                            int32_t u_max, int32_t* q_out, int32_t* U_out)
{
    if (nb < 1 || window < 1 || alpha_ppm <= 0 || alpha_ppm >= 1000000 || n < 0 || m < 0) return -1;
    for (int64_t i = 0; i < n; ++i)
        if (pred[i] < 0 || truth[i] < 0) return -4;
    /* where each bucket's completions sit in the log, in log order */
    int64_t* count = (int64_t*)calloc((size_t)nb, sizeof(int64_t));
    int64_t* start = (int64_t*)calloc((size_t)nb + 1, sizeof(int64_t));
    int64_t* fill = (int64_t*)calloc((size_t)nb, sizeof(int64_t));
    int64_t* pos = (int64_t*)malloc((size_t)(n > 0 ? n : 1) * sizeof(int64_t));
    int64_t* set = (int64_t*)malloc((size_t)window * sizeof(int64_t));
    if (!count || !start || !fill || !pos || !set) return -2;
    for (int64_t i = 0; i < n; ++i) count[oracle_bucket(pred[i], edges, nb)] += 1;
    for (int32_t b = 0; b < nb; ++b) start[b + 1] = start[b] + count[b];
    for (int64_t i = 0; i < n; ++i) {
        int32_t b = oracle_bucket(pred[i], edges, nb);
        pos[start[b] + fill[b]] = i;
        fill[b] += 1;
    }
    int rc = 0;
    for (int64_t j = 0; j < m; ++j) {
        if (apply_pred[j] < 0) { q_out[j] = -1; U_out[j] = -1; continue; }
        if (seen[j] < 0 || seen[j] > n) { rc = -3; break; }
        int32_t b = oracle_bucket(apply_pred[j], edges, nb);
        /* c = completions of bucket b logged before entry seen[j] */
        int64_t lo = 0, hi = count[b];
        while (lo < hi) {
            int64_t mid = lo + (hi - lo) / 2;
            if (pos[start[b] + mid] < seen[j]) lo = mid + 1; else hi = mid;
        }
        int64_t c = lo;
        int64_t nw = min64(c, window);
        /* the set: the last nw of them; Eq. (2) scores */
        for (int64_t t = 0; t < nw; ++t) {
            int64_t i = pos[start[b] + c - nw + t];
            set[t] = max64(0, (int64_t)truth[i] - (int64_t)pred[i]);
        }
        qsort(set, (size_t)nw, sizeof(int64_t), cmp_i64);
        int64_t k = oracle_conformal_rank(nw, alpha_ppm);
        int32_t q = (k <= nw) ? (int32_t)set[k - 1] : ORACLE_Q_INF;
        q_out[j] = q;
        if (q == ORACLE_Q_INF) U_out[j] = u_max;
        else U_out[j] = (int32_t)min64((int64_t)apply_pred[j] + q, u_max);
    }
    free(count); free(start); free(fill); free(pos); free(set);
    return rc;
}

/* ------------------------------------------------------------------------ */
/* Occupancy, one decoding step at a time (Sec. 3.3, App. A)                 */
/* ------------------------------------------------------------------------ */

static int64_t remaining(int32_t U, int32_t g) { return max64((int64_t)U - g, 0); }

/* O[t], t = 0..T: total KV tokens held at step t by the residents still
 * decoding.  Each resident holds p+g+t and leaves after step R. */
int oracle_occupancy(const int32_t* p, const int32_t* g, const int32_t* U, int64_t n,
                     int64_t T, int64_t* O)
{
    int64_t* leave_cnt = (int64_t*)calloc((size_t)T + 1, sizeof(int64_t));
    int64_t* leave_tok = (int64_t*)calloc((size_t)T + 1, sizeof(int64_t));
    if (!leave_cnt || !leave_tok) return -2;
    int64_t active = 0, held = 0;   /* requests decoding, and their p+g */
    for (int64_t r = 0; r < n; ++r) {
        if (p[r] < 0 || g[r] < 0 || U[r] < 0) { free(leave_cnt); free(leave_tok); return -1; }
        int64_t R = remaining(U[r], g[r]);
        if (R > T) { free(leave_cnt); free(leave_tok); return -3; }
        active += 1;
        held += (int64_t)p[r] + g[r];
        leave_cnt[R] += 1;
        leave_tok[R] += (int64_t)p[r] + g[r];
    }
    for (int64_t t = 0; t <= T; ++t) {
        O[t] = held + t * active;      /* every active request holds p+g+t */
        active -= leave_cnt[t];        /* those whose last step is t leave */
        held -= leave_tok[t];
    }
    free(leave_cnt); free(leave_tok);
    return 0;
}

static int64_t max_remaining(const int32_t* g, const int32_t* U, int64_t lo, int64_t hi)
{
    int64_t T = 0;
    for (int64_t r = lo; r < hi; ++r) T = max64(T, remaining(U[r], g[r]));
    return T;
}

/* Peak of the projected occupancy of each decoder on its own. */
int oracle_project(int32_t D, const int64_t* seg_off, const int32_t* p, const int32_t* g,
                   const int32_t* U, int64_t* base_peak)
{
    for (int32_t d = 0; d < D; ++d) {
        int64_t lo = seg_off[d], hi = seg_off[d + 1];
        int64_t T = max_remaining(g, U, lo, hi);
        int64_t* O = (int64_t*)malloc(((size_t)T + 1) * sizeof(int64_t));
        if (!O) return -2;
        int rc = oracle_occupancy(p + lo, g + lo, U + lo, hi - lo, T, O);
        if (rc) { free(O); return rc; }
        int64_t peak = 0;
        for (int64_t t = 0; t <= T; ++t) peak = max64(peak, O[t]);
        base_peak[d] = peak;
        free(O);
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Placement (Algorithm 1 with the projected peak as the feasibility test)   */
/* ------------------------------------------------------------------------ */

/*
 * For every arrival a and decoder d:
 *   peak(a, d) = max_t [ O_d[t] + (t <= U_a ? p_a + t : 0) ]
 * taken over the dense step axis.  The maximum splits at U_a into the steps the
 * arrival is present (t <= U_a, where it adds p_a + t) and the later ones, so
 *   peak = max( p_a + max_{t<=U_a} (O[t] + t),  max_{t>U_a} O[t] ).
 * slack = C_d - peak.  Choice (policy MQ): among decoders with slack >= 0 the
 * smallest queue length Q_d; when there is none, the largest slack.  Policy MC:
 * the largest slack.  Ties go to the lowest index.  A negative bound routes
 * the arrival round-robin: d = (rr_offset + i) mod D, i its arrival index.
 *
 * pair_peak (nullable) is decoder-major [D][A]; -1 for round-robin arrivals.
 * a_index (nullable) gives each arrival's index for the round-robin rule.
 */
int oracle_place(int32_t D, const int64_t* seg_off, const int32_t* p, const int32_t* g,
                 const int32_t* U, const int32_t* capacity, const int32_t* queue_len,
                 int64_t A, const int32_t* a_p, const int32_t* a_U, const int64_t* a_index,
                 int32_t policy, int64_t rr_offset,
                 int32_t* choice, int64_t* chosen_peak, int64_t* chosen_overflow,
                 uint8_t* flags, int64_t* pair_peak, int64_t* base_peak)
{
    if (D < 1 || A < 0 || (policy != ORACLE_POLICY_MQ && policy != ORACLE_POLICY_MC)) return -1;
    int64_t maxU = 0;
    for (int64_t a = 0; a < A; ++a) maxU = max64(maxU, a_U[a]);

    int32_t* feas_d = (int32_t*)malloc((size_t)(A > 0 ? A : 1) * sizeof(int32_t));
    int64_t* feas_peak = (int64_t*)malloc((size_t)(A > 0 ? A : 1) * sizeof(int64_t));
    int32_t* fb_d = (int32_t*)malloc((size_t)(A > 0 ? A : 1) * sizeof(int32_t));
    int64_t* fb_slack = (int64_t*)malloc((size_t)(A > 0 ? A : 1) * sizeof(int64_t));
    int64_t* fb_peak = (int64_t*)malloc((size_t)(A > 0 ? A : 1) * sizeof(int64_t));
    if (!feas_d || !feas_peak || !fb_d || !fb_slack || !fb_peak) return -2;
    for (int64_t a = 0; a < A; ++a) { feas_d[a] = -1; fb_d[a] = -1; }

    for (int32_t d = 0; d < D; ++d) {
        int64_t lo = seg_off[d], hi = seg_off[d + 1];
        int64_t T = max64(max_remaining(g, U, lo, hi), maxU);
        int64_t* O = (int64_t*)malloc(((size_t)T + 1) * sizeof(int64_t));
        int64_t* present = (int64_t*)malloc(((size_t)T + 1) * sizeof(int64_t));
        int64_t* after = (int64_t*)malloc(((size_t)T + 1) * sizeof(int64_t));
        if (!O || !present || !after) return -2;
        int rc = oracle_occupancy(p + lo, g + lo, U + lo, hi - lo, T, O);
        if (rc) return rc;
        int64_t peak0 = 0;
        for (int64_t t = 0; t <= T; ++t) peak0 = max64(peak0, O[t]);
        if (base_peak) base_peak[d] = peak0;
        /* present[u] = max_{t<=u} (O[t] + t);  after[u] = max_{t>u} O[t] */
        for (int64_t t = 0; t <= T; ++t)
            present[t] = (t == 0) ? O[0] : max64(present[t - 1], O[t] + t);
        after[T] = 0;                      /* O[t] = 0 beyond T */
        for (int64_t t = T - 1; t >= 0; --t) after[t] = max64(after[t + 1], O[t + 1]);

        for (int64_t a = 0; a < A; ++a) {
            if (a_U[a] < 0) {
                if (pair_peak) pair_peak[(int64_t)d * A + a] = -1;
                continue;
            }
            int64_t peak = max64((int64_t)a_p[a] + present[a_U[a]], after[a_U[a]]);
            int64_t slack = (int64_t)capacity[d] - peak;
            if (pair_peak) pair_peak[(int64_t)d * A + a] = peak;
            if (policy == ORACLE_POLICY_MQ && slack >= 0) {
                if (feas_d[a] < 0 || queue_len[d] < queue_len[feas_d[a]]) {
                    feas_d[a] = d;
                    feas_peak[a] = peak;
                }
            }
            if (fb_d[a] < 0 || slack > fb_slack[a]) {
                fb_d[a] = d;
                fb_slack[a] = slack;
                fb_peak[a] = peak;
            }
        }
        free(O); free(present); free(after);
    }

    for (int64_t a = 0; a < A; ++a) {
        if (a_U[a] < 0) {
            int64_t i = a_index ? a_index[a] : a;
            choice[a] = (int32_t)((rr_offset + i) % D);
            chosen_peak[a] = -1;
            chosen_overflow[a] = 0;
            flags[a] = 2;
        } else if (policy == ORACLE_POLICY_MQ && feas_d[a] >= 0) {
            choice[a] = feas_d[a];
            chosen_peak[a] = feas_peak[a];
            chosen_overflow[a] = 0;
            flags[a] = 1;
        } else {
            int64_t c = capacity[fb_d[a]];
            choice[a] = fb_d[a];
            chosen_peak[a] = fb_peak[a];
            chosen_overflow[a] = max64(0, fb_peak[a] - c);
            flags[a] = (fb_peak[a] <= c) ? 1 : 0;
        }
    }
    free(feas_d); free(feas_peak); free(fb_d); free(fb_slack); free(fb_peak);
    return 0;
}

/*
 * Placement with sequential commit (Sec. 3.3: each dispatch atomically
 * reserves its demand before the next request is placed; Algorithm 1).
 * Arrivals are taken in index order.  Arrival a is evaluated exactly as in
 * oracle_place, but against occupancy curves that include every earlier
 * arrival already committed to the decoder: a committed arrival (p, U) holds
 * p + t at step t while t <= U (a resident with g = 0 and R = U).  The chosen
 * decoder then receives the arrival (its curve grows by p + t for t <= U) and
 * its queue grows by one; the queue lengths that MQ compares are these
 * running ones.  An arrival without a bound goes round robin, joins that
 * decoder's queue and commits no occupancy (its footprint is unknown).
 * queue_out (nullable) receives the queue lengths after the batch.
 */
int oracle_place_commit(int32_t D, const int64_t* seg_off, const int32_t* p, const int32_t* g,
                        const int32_t* U, const int32_t* capacity, const int32_t* queue_len,
                        int64_t A, const int32_t* a_p, const int32_t* a_U, int32_t policy, int64_t rr_offset,
                        int32_t* choice, int64_t* chosen_peak, int64_t* chosen_overflow, uint8_t* flags,
                        int32_t* queue_out)
{
    if (D < 1 || A < 0 || rr_offset < 0 || (policy != ORACLE_POLICY_MQ && policy != ORACLE_POLICY_MC)) return -1;
    int64_t T = 0;
    for (int64_t a = 0; a < A; ++a) T = max64(T, a_U[a]);
    for (int32_t d = 0; d < D; ++d) T = max64(T, max_remaining(g, U, seg_off[d], seg_off[d + 1]));
    size_t len = (size_t)T + 1;
    /* per decoder: the occupancy curve O, present[u] = max_{t<=u} (O[t] + t)
     * and after[u] = max_{t>u} O[t] (0 past T), as in oracle_place */
    int64_t* O = (int64_t*)malloc((size_t)D * len * sizeof(int64_t));
    int64_t* present = (int64_t*)malloc((size_t)D * len * sizeof(int64_t));
    int64_t* after = (int64_t*)malloc((size_t)D * len * sizeof(int64_t));
    int64_t* Q = (int64_t*)malloc((size_t)D * sizeof(int64_t));
    if (!O || !present || !after || !Q) { free(O); free(present); free(after); free(Q); return -2; }
    int rc = 0;
    for (int32_t d = 0; d < D && rc == 0; ++d) {
        int64_t lo = seg_off[d], hi = seg_off[d + 1];
        rc = oracle_occupancy(p + lo, g + lo, U + lo, hi - lo, T, O + (size_t)d * len);
        Q[d] = queue_len[d];
    }
    for (int32_t d = 0; d < D && rc == 0; ++d) {   /* the derived maxima of every decoder */
        int64_t *o = O + (size_t)d * len, *pr = present + (size_t)d * len, *af = after + (size_t)d * len;
        for (int64_t t = 0; t <= T; ++t) pr[t] = (t == 0) ? o[0] : max64(pr[t - 1], o[t] + t);
        af[T] = 0;
        for (int64_t t = T - 1; t >= 0; --t) af[t] = max64(af[t + 1], o[t + 1]);
    }
    for (int64_t a = 0; a < A && rc == 0; ++a) {
        if (a_U[a] < 0) {
            int32_t d = (int32_t)((rr_offset + a) % D);
            choice[a] = d;
            chosen_peak[a] = -1;
            chosen_overflow[a] = 0;
            flags[a] = 2;
            Q[d] += 1;
            continue;
        }
        int32_t feas_d = -1, fb_d = -1;
        int64_t feas_peak = 0, fb_slack = 0, fb_peak = 0;
        for (int32_t d = 0; d < D; ++d) {
            int64_t peak = max64((int64_t)a_p[a] + present[(size_t)d * len + a_U[a]], after[(size_t)d * len + a_U[a]]);
            int64_t slack = (int64_t)capacity[d] - peak;
            if (policy == ORACLE_POLICY_MQ && slack >= 0 && (feas_d < 0 || Q[d] < Q[feas_d])) {
                feas_d = d;
                feas_peak = peak;
            }
            if (fb_d < 0 || slack > fb_slack) {
                fb_d = d;
                fb_slack = slack;
                fb_peak = peak;
            }
        }
        int32_t best;
        if (policy == ORACLE_POLICY_MQ && feas_d >= 0) {
            best = feas_d;
            chosen_peak[a] = feas_peak;
            chosen_overflow[a] = 0;
            flags[a] = 1;
        } else {
            best = fb_d;
            chosen_peak[a] = fb_peak;
            chosen_overflow[a] = max64(0, fb_peak - capacity[fb_d]);
            flags[a] = (fb_peak <= capacity[fb_d]) ? 1 : 0;
        }
        choice[a] = best;
        Q[best] += 1;
        /* commit: the arrival joins the chosen decoder's curve, whose maxima
         * are then derived again over the whole step axis */
        int64_t *o = O + (size_t)best * len, *pr = present + (size_t)best * len, *af = after + (size_t)best * len;
        for (int64_t t = 0; t <= a_U[a]; ++t) o[t] += (int64_t)a_p[a] + t;
        for (int64_t t = 0; t <= T; ++t) pr[t] = (t == 0) ? o[0] : max64(pr[t - 1], o[t] + t);
        af[T] = 0;
        for (int64_t t = T - 1; t >= 0; --t) af[t] = max64(af[t + 1], o[t + 1]);
    }
    if (rc == 0 && queue_out)
        for (int32_t d = 0; d < D; ++d) queue_out[d] = (int32_t)Q[d];
    free(O); free(present); free(after); free(Q);
    return rc;
}

/* ------------------------------------------------------------------------ */
/* Algorithm 1 on block counts (Sec. 3.3: the runtime state, Eq. (6),        */
/* Algorithm 1 and the atomic reservation of B_need after each dispatch)      */
/* ------------------------------------------------------------------------ */

static int64_t ceil_div(int64_t x, int64_t s) { return (x + s - 1) / s; }

/* Runtime state of each decoder in blocks of S tokens: capacity floor(C/S)
 * blocks; each resident holds ceil((p+g)/S) blocks and keeps reserved the
 * blocks still missing to its demand ceil((p+U)/S) (none when U < 0 or when
 * it already holds more); B_free = capacity blocks - held blocks,
 * B_res = sum of the reservations, B_eff = B_free - B_res.  in_flight
 * (nullable) marks requests whose prompt KV is still in transfer. */
int oracle_rsc_state(int32_t D, const int64_t* seg_off, const int32_t* p, const int32_t* g,
                     const int32_t* U, const uint8_t* in_flight, const int32_t* capacity, int32_t S,
                     int64_t* b_free, int64_t* b_res, int64_t* b_eff)
{
    if (D < 1 || S < 1) return -1;
    for (int32_t d = 0; d < D; ++d) {
        int64_t held = 0, res = 0;
        for (int64_t r = seg_off[d]; r < seg_off[d + 1]; ++r) {
            if (in_flight && in_flight[r]) {
                /* Staged reservation (appendix on the global algorithm): a request
                 * dispatched here whose prompt KV has not arrived yet holds no
                 * block and keeps its whole budget reserved, ceil((p+U)/S) (its
                 * prompt's blocks when it has no bound).  Once the prompt is
                 * transferred the prompt part of that reservation is released
                 * into held blocks, the rule below. */
                res += U[r] < 0 ? ceil_div((int64_t)p[r], S) : ceil_div((int64_t)p[r] + U[r], S);
                continue;
            }
            int64_t now = ceil_div((int64_t)p[r] + g[r], S);
            int64_t demand = U[r] < 0 ? now : ceil_div((int64_t)p[r] + U[r], S);
            held += now;
            res += max64(demand - now, 0);
        }
        b_free[d] = (int64_t)capacity[d] / S - held;
        b_res[d] = res;
        b_eff[d] = b_free[d] - res;
    }
    return 0;
}

/* Algorithm 1 for A arrivals in order: B_need = ceil((p+U)/S) (Eq. (6)); the
 * feasible decoders have B_need <= B_eff; policy MQ takes the feasible one
 * with the shortest queue (lowest index on ties), else the largest B_eff
 * (lowest index on ties); policy MC always the largest B_eff.  An arrival
 * without a bound (U < 0) goes round robin, (rr_offset + a) mod D, with
 * b_need -1.  With reserve != 0 each dispatch then reserves its B_need on the
 * chosen decoder and joins its queue (B_eff -= B_need, Q += 1; a round-robin
 * dispatch only joins the queue), so later arrivals see the new state; with
 * reserve == 0 every arrival sees the given state.  flags: bit0 when B_need <=
 * B_eff of the chosen decoder (before its reservation), bit1 round robin.
 * b_eff_out / q_out (if not NULL) receive the state after the batch. */
int oracle_place_static(int32_t D, const int64_t* b_eff_in, const int32_t* queue_len, int32_t S,
                        int64_t A, const int32_t* a_p, const int32_t* a_U, int32_t policy,
                        int64_t rr_offset, int32_t reserve, int32_t* choice, int64_t* b_need,
                        uint8_t* flags, int64_t* b_eff_out, int32_t* q_out)
{
    if (D < 1 || A < 0 || S < 1 || rr_offset < 0 ||
        (policy != ORACLE_POLICY_MQ && policy != ORACLE_POLICY_MC)) return -1;
    int64_t* B = (int64_t*)malloc((size_t)D * sizeof(int64_t));
    int64_t* Q = (int64_t*)malloc((size_t)D * sizeof(int64_t));
    if (!B || !Q) return -2;
    for (int32_t d = 0; d < D; ++d) { B[d] = b_eff_in[d]; Q[d] = queue_len[d]; }
    for (int64_t a = 0; a < A; ++a) {
        int32_t best;
        if (a_U[a] < 0) {
            best = (int32_t)((rr_offset + a) % D);
            choice[a] = best;
            b_need[a] = -1;
            flags[a] = 2;
            if (reserve) Q[best] += 1;
            continue;
        }
        int64_t need = ceil_div((int64_t)a_p[a] + a_U[a], S);
        int32_t feas = -1, most = 0;
        for (int32_t d = 0; d < D; ++d) {
            if (need <= B[d] && (feas < 0 || Q[d] < Q[feas])) feas = d;
            if (B[d] > B[most]) most = d;
        }
        best = (policy == ORACLE_POLICY_MQ && feas >= 0) ? feas : most;
        choice[a] = best;
        b_need[a] = need;
        flags[a] = (uint8_t)(need <= B[best] ? 1 : 0);
        if (reserve) { B[best] -= need; Q[best] += 1; }
    }
    for (int32_t d = 0; d < D; ++d) {
        if (b_eff_out) b_eff_out[d] = B[d];
        if (q_out) q_out[d] = (int32_t)Q[d];
    }
    free(B); free(Q);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Projected peak in blocks (Sec. 3.3: capacity in blocks of S tokens;       */
/* Eq. (6) counts a request's blocks as ceil(tokens / S))                    */
/* ------------------------------------------------------------------------ */

/* OB[t], t = 0..T: KV blocks held at step t by the residents still decoding,
 * each holding ceil((p+g+t)/S) blocks while t <= R.  Step by step: from t to
 * t+1 a request gains a block exactly when p+g+t is a multiple of S, and the
 * requests whose last step is t leave with their blocks. */
int oracle_occupancy_blocks(const int32_t* p, const int32_t* g, const int32_t* U, int64_t n,
                            int32_t S, int64_t T, int64_t* OB)
{
    int64_t* leave_first = (int64_t*)malloc(((size_t)T + 2) * sizeof(int64_t));
    int64_t* next = (int64_t*)malloc((size_t)(n > 0 ? n : 1) * sizeof(int64_t));
    int64_t* active_in = (int64_t*)calloc((size_t)S, sizeof(int64_t));   /* active requests by (p+g) mod S */
    if (!leave_first || !next || !active_in) return -2;
    for (int64_t t = 0; t <= T + 1; ++t) leave_first[t] = -1;
    int64_t held = 0;
    for (int64_t r = 0; r < n; ++r) {
        if (p[r] < 0 || g[r] < 0 || U[r] < 0) { free(leave_first); free(next); free(active_in); return -1; }
        int64_t R = remaining(U[r], g[r]);
        if (R > T) { free(leave_first); free(next); free(active_in); return -3; }
        int64_t x = (int64_t)p[r] + g[r];
        held += (x + S - 1) / S;                 /* blocks at step 0 */
        active_in[x % S] += 1;
        next[r] = leave_first[R];                /* requests leaving after step R */
        leave_first[R] = r;
    }
    for (int64_t t = 0; t <= T; ++t) {
        OB[t] = held;
        for (int64_t r = leave_first[t]; r >= 0; r = next[r]) {
            int64_t x = (int64_t)p[r] + g[r];
            held -= (x + t + S - 1) / S;
            active_in[x % S] -= 1;
        }
        /* the requests still active gain a block when p+g+t = 0 mod S */
        held += active_in[(S - t % S) % S];
    }
    free(leave_first); free(next); free(active_in);
    return 0;
}

/* Placement in blocks: peak(a, d) = max_t [OB_d[t] + [t <= U_a] ceil((p_a+t)/S)],
 * capacity floor(C_d / S) blocks; the choice as in oracle_place. */
int oracle_place_blocks(int32_t D, const int64_t* seg_off, const int32_t* p, const int32_t* g,
                        const int32_t* U, const int32_t* capacity, const int32_t* queue_len, int32_t S,
                        int64_t A, const int32_t* a_p, const int32_t* a_U, int32_t policy, int64_t rr_offset,
                        int32_t* choice, int64_t* chosen_peak, int64_t* chosen_overflow,
                        uint8_t* flags, int64_t* pair_peak, int64_t* base_peak)
{
    if (D < 1 || A < 0 || S < 1 || (policy != ORACLE_POLICY_MQ && policy != ORACLE_POLICY_MC)) return -1;
    int64_t maxU = 0;
    for (int64_t a = 0; a < A; ++a) maxU = max64(maxU, a_U[a]);
    int32_t* feas_d = (int32_t*)malloc((size_t)(A > 0 ? A : 1) * sizeof(int32_t));
    int64_t* feas_peak = (int64_t*)malloc((size_t)(A > 0 ? A : 1) * sizeof(int64_t));
    int32_t* fb_d = (int32_t*)malloc((size_t)(A > 0 ? A : 1) * sizeof(int32_t));
    int64_t* fb_slack = (int64_t*)malloc((size_t)(A > 0 ? A : 1) * sizeof(int64_t));
    int64_t* fb_peak = (int64_t*)malloc((size_t)(A > 0 ? A : 1) * sizeof(int64_t));
    if (!feas_d || !feas_peak || !fb_d || !fb_slack || !fb_peak) return -2;
    for (int64_t a = 0; a < A; ++a) { feas_d[a] = -1; fb_d[a] = -1; }

    for (int32_t d = 0; d < D; ++d) {
        int64_t lo = seg_off[d], hi = seg_off[d + 1];
        int64_t T = max64(max_remaining(g, U, lo, hi), maxU);
        int64_t* OB = (int64_t*)malloc(((size_t)T + 1) * sizeof(int64_t));
        int64_t* present = (int64_t*)malloc((size_t)S * ((size_t)T + 1) * sizeof(int64_t));
        int64_t* after = (int64_t*)malloc(((size_t)T + 1) * sizeof(int64_t));
        if (!OB || !present || !after) return -2;
        int rc = oracle_occupancy_blocks(p + lo, g + lo, U + lo, hi - lo, S, T, OB);
        if (rc) return rc;
        int64_t peak0 = 0;
        for (int64_t t = 0; t <= T; ++t) peak0 = max64(peak0, OB[t]);
        if (base_peak) base_peak[d] = peak0;
        /* present[rho][u] = max_{t<=u} (OB[t] + ceil((rho+t)/S));  after[u] = max_{t>u} OB[t] */
        for (int32_t rho = 0; rho < S; ++rho) {
            int64_t* pr = present + (size_t)rho * ((size_t)T + 1);
            for (int64_t t = 0; t <= T; ++t) {
                int64_t v = OB[t] + (rho + t + S - 1) / S;
                pr[t] = (t == 0) ? v : max64(pr[t - 1], v);
            }
        }
        after[T] = 0;
        for (int64_t t = T - 1; t >= 0; --t) after[t] = max64(after[t + 1], OB[t + 1]);
        int64_t capB = (int64_t)capacity[d] / S;

        for (int64_t a = 0; a < A; ++a) {
            if (a_U[a] < 0) {
                if (pair_peak) pair_peak[(int64_t)d * A + a] = -1;
                continue;
            }
            /* ceil((p+t)/S) = p div S + ceil((p mod S + t)/S) */
            int64_t P = a_p[a] / S, rho = a_p[a] % S;
            int64_t peak = max64(P + present[(size_t)rho * ((size_t)T + 1) + a_U[a]], after[a_U[a]]);
            int64_t slack = capB - peak;
            if (pair_peak) pair_peak[(int64_t)d * A + a] = peak;
            if (policy == ORACLE_POLICY_MQ && slack >= 0) {
                if (feas_d[a] < 0 || queue_len[d] < queue_len[feas_d[a]]) {
                    feas_d[a] = d;
                    feas_peak[a] = peak;
                }
            }
            if (fb_d[a] < 0 || slack > fb_slack[a]) {
                fb_d[a] = d;
                fb_slack[a] = slack;
                fb_peak[a] = peak;
            }
        }
        free(OB); free(present); free(after);
    }

    for (int64_t a = 0; a < A; ++a) {
        if (a_U[a] < 0) {
            choice[a] = (int32_t)((rr_offset + a) % D);
            chosen_peak[a] = -1;
            chosen_overflow[a] = 0;
            flags[a] = 2;
        } else if (policy == ORACLE_POLICY_MQ && feas_d[a] >= 0) {
            choice[a] = feas_d[a];
            chosen_peak[a] = feas_peak[a];
            chosen_overflow[a] = 0;
            flags[a] = 1;
        } else {
            int64_t c = (int64_t)capacity[fb_d[a]] / S;
            choice[a] = fb_d[a];
            chosen_peak[a] = fb_peak[a];
            chosen_overflow[a] = max64(0, fb_peak[a] - c);
            flags[a] = (fb_peak[a] <= c) ? 1 : 0;
        }
    }
    free(feas_d); free(feas_peak); free(fb_d); free(fb_slack); free(fb_peak);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Local order and admission (Sec. 3.3, Eq. (7); App. A, Eq. (10))           */
/* ------------------------------------------------------------------------ */

typedef struct {
    int64_t cls;    /* 0: promoted past the maximum wait, 1: otherwise */
    int64_t val;    /* promoted: queue index (FCFS); otherwise the bound */
    int64_t idx;    /* queue index, the final tie-break */
} order_key;

static int cmp_key(const void* a, const void* b)
{
    const order_key* x = (const order_key*)a;
    const order_key* y = (const order_key*)b;
    if (x->cls != y->cls) return x->cls < y->cls ? -1 : 1;
    if (x->val != y->val) return x->val < y->val ? -1 : 1;
    if (x->idx != y->idx) return x->idx < y->idx ? -1 : 1;
    return 0;
}

/*
 * Per decoder: order the pending queue by its bounds (Eq. (7)); requests that
 * waited at least max_wait_ms go first, in arrival order; equal bounds keep
 * arrival order.  A missing bound (< 0) counts as u_max.  Then admit requests
 * in that order while the projected peak of the residents plus the admitted
 * requests (each starting now, g = 0) stays within the capacity: admitted[d]
 * is the length of that prefix.  order holds queue-local indices.
 */
int oracle_local_order(int32_t D, const int64_t* seg_off, const int32_t* p, const int32_t* g,
                       const int32_t* U, const int32_t* capacity, const int64_t* q_off,
                       const int32_t* q_p, const int32_t* q_U, const int32_t* q_wait,
                       int32_t max_wait_ms, int32_t u_max, int32_t* order, int32_t* admitted)
{
    for (int32_t d = 0; d < D; ++d) {
        int64_t qlo = q_off[d], nq = q_off[d + 1] - q_off[d];
        order_key* keys = (order_key*)malloc((size_t)(nq > 0 ? nq : 1) * sizeof(order_key));
        if (!keys) return -2;
        int64_t maxU = 0;
        for (int64_t i = 0; i < nq; ++i) {
            int64_t Ui = q_U[qlo + i] < 0 ? u_max : q_U[qlo + i];
            int promoted = q_wait != NULL && q_wait[qlo + i] >= max_wait_ms;
            keys[i].cls = promoted ? 0 : 1;
            keys[i].val = promoted ? i : Ui;
            keys[i].idx = i;
            maxU = max64(maxU, Ui);
        }
        qsort(keys, (size_t)nq, sizeof(order_key), cmp_key);
        for (int64_t i = 0; i < nq; ++i) order[qlo + i] = (int32_t)keys[i].idx;

        int64_t lo = seg_off[d], hi = seg_off[d + 1];
        int64_t T = max64(max_remaining(g, U, lo, hi), maxU);
        int64_t* G = (int64_t*)malloc(((size_t)T + 1) * sizeof(int64_t));
        if (!G) return -2;
        int rc = oracle_occupancy(p + lo, g + lo, U + lo, hi - lo, T, G);
        if (rc) return rc;
        int64_t peak = 0;
        for (int64_t t = 0; t <= T; ++t) peak = max64(peak, G[t]);
        int64_t k = 0;
        if (peak <= capacity[d]) {
            for (; k < nq; ++k) {
                int64_t i = keys[k].idx;
                int64_t Ui = q_U[qlo + i] < 0 ? u_max : q_U[qlo + i];
                for (int64_t t = 0; t <= Ui; ++t) {
                    G[t] += (int64_t)q_p[qlo + i] + t;
                    peak = max64(peak, G[t]);
                }
                if (peak > capacity[d]) break;
            }
        }
        admitted[d] = (int32_t)k;
        free(G); free(keys);
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Brute force (tiny inputs only)                                            */
/* ------------------------------------------------------------------------ */

/* max over t of  sum_r [t <= R_r] (p_r + g_r + t)  +  sum_k [t <= V_k] (q_k + t),
 * evaluated term by term at every step t up to the last one anything is held. */
int64_t oracle_bruteforce_peak(int64_t n, const int32_t* p, const int32_t* g, const int32_t* U,
                               int64_t m, const int32_t* q, const int32_t* V)
{
    int64_t T = 0;
    for (int64_t r = 0; r < n; ++r) T = max64(T, remaining(U[r], g[r]));
    for (int64_t k = 0; k < m; ++k) T = max64(T, V[k]);
    int64_t best = 0;
    for (int64_t t = 0; t <= T; ++t) {
        int64_t occ = 0;
        for (int64_t r = 0; r < n; ++r)
            if (t <= remaining(U[r], g[r])) occ += (int64_t)p[r] + g[r] + t;
        for (int64_t k = 0; k < m; ++k)
            if (t <= V[k]) occ += (int64_t)q[k] + t;
        best = max64(best, occ);
    }
    return best;
}

/* ------------------------------------------------------------------------ */
/* App. A: KV pressure of decoders under round-robin or MAPS routing,        */
/* simulated one decoding step (t_tok = 1 ms) at a time                      */
/* ------------------------------------------------------------------------ */

/*
 * N decoders with a KV capacity of C tokens each serve n requests taken in
 * arrival order (arrival_ms non-decreasing, whole milliseconds).  Request i
 * has prompt L_p = prompt[i] >= 0, output L_out = output[i] >= 1 and KV demand
 * M = L_p + L_out (Eq. (8)), held from its admission to its completion.
 * Routing: policy 0 is round robin, d = i mod N (Eq. (9), decoders counted
 * from 0).  Policy 1 is Algorithm 1 at block size 1 on the decoders' state:
 * B_need = L_p + bound[i]; B_eff(d) = C - K_d - (the needs of the requests
 * waiting in d's queue, reserved when they were dispatched); Q_d the length of
 * d's queue; the feasible decoder (B_need <= B_eff) with the shortest queue,
 * else the largest B_eff, lowest index on ties; a request without a bound
 * (bound < 0) goes round robin.
 *
 * Every millisecond t, in this order:
 *   1. the request whose last token a decoder decoded during [t-1, t)
 *      completes at t and releases its M tokens;
 *   2. every decoder admits the head of its FIFO queue while K_d + M <= C
 *      (Eq. (10)), again and again;
 *   3. the requests arriving at t are routed in index order; a request is
 *      admitted at once when its decoder's queue is empty and K_d + M <= C,
 *      else it joins the queue;
 *   4. the state for [t, t+1) is recorded: decoder d is under high pressure
 *      when K_d / C >= theta (the HP interval definition), and its queue
 *      length is added up;
 *   5. every decoder decodes one token of the request at the head of its
 *      ready queue (processor sharing by time slices of one token: one token
 *      per t_tok in total, the admitted requests in turn); a request with
 *      tokens left goes to the back of the ready queue, and a newly admitted
 *      request joins it at the back.
 * Outputs: finish_ms[i], routed[i]; per decoder hp_time (milliseconds under
 * pressure within [first arrival, last completion)), hp_max (longest
 * pressure interval), hp_count (number of intervals), max_queue and
 * queue_area (sum over milliseconds of the queue length); span[0] = first
 * arrival, span[1] = last completion.  theta is theta_ppm / 10^6.
 * Returns -1 for invalid arguments, M > C or L_out < 1 in a request.
 */
int oracle_simulate(int32_t N, int64_t C, int32_t theta_ppm, int64_t n, const int64_t* arrival_ms,
                    const int32_t* prompt, const int32_t* output, const int32_t* bound, int32_t policy,
                    int64_t* finish_ms, int32_t* routed, int64_t* hp_time, int64_t* hp_max, int64_t* hp_count,
                    int64_t* max_queue, int64_t* queue_area, int64_t* span)
{
    if (N < 1 || C < 1 || n < 1 || theta_ppm < 1 || theta_ppm > 1000000 || (policy != 0 && policy != 1)) return -1;
    for (int64_t i = 0; i < n; ++i) {
        if (prompt[i] < 0 || output[i] < 1 || (int64_t)prompt[i] + output[i] > C) return -1;
        if (i > 0 && arrival_ms[i] < arrival_ms[i - 1]) return -1;
    }
    /* per decoder: the ready queue and the FIFO queue as plain arrays of
     * request indices (front at index 0, shifted on removal) */
    int64_t* ready = (int64_t*)malloc((size_t)N * n * sizeof(int64_t));
    int64_t* fifo = (int64_t*)malloc((size_t)N * n * sizeof(int64_t));
    int64_t* nready = (int64_t*)calloc((size_t)N, sizeof(int64_t));
    int64_t* nfifo = (int64_t*)calloc((size_t)N, sizeof(int64_t));
    int64_t* K = (int64_t*)calloc((size_t)N, sizeof(int64_t));
    int64_t* R = (int64_t*)calloc((size_t)N, sizeof(int64_t));
    int64_t* release = (int64_t*)malloc((size_t)N * sizeof(int64_t));
    int64_t* run = (int64_t*)calloc((size_t)N, sizeof(int64_t));
    int64_t* left = (int64_t*)malloc((size_t)n * sizeof(int64_t));
    if (!ready || !fifo || !nready || !nfifo || !K || !R || !release || !run || !left) {
        free(ready); free(fifo); free(nready); free(nfifo); free(K); free(R); free(release); free(run); free(left);
        return -2;
    }
    for (int32_t d = 0; d < N; ++d) {
        release[d] = -1;
        hp_time[d] = hp_max[d] = hp_count[d] = max_queue[d] = queue_area[d] = 0;
    }
    for (int64_t i = 0; i < n; ++i) left[i] = output[i];
#define DEMAND(i) ((int64_t)prompt[i] + output[i])
#define NEED(i) ((int64_t)prompt[i] + bound[i])
    int64_t t = arrival_ms[0], next = 0, done = 0;
    span[0] = t;
    span[1] = t;
    for (;;) {
        /* 1. completions */
        for (int32_t d = 0; d < N; ++d) {
            if (release[d] < 0) continue;
            K[d] -= DEMAND(release[d]);
            finish_ms[release[d]] = t;
            release[d] = -1;
            done += 1;
            span[1] = t;
        }
        if (done == n) break;
        /* a stretch with nothing admitted, queued or arriving: every decoder
         * idle (no pressure, empty queues) until the next arrival */
        int idle = 1;
        for (int32_t d = 0; d < N; ++d) if (nready[d] || nfifo[d]) idle = 0;
        if (idle && next < n && arrival_ms[next] > t) {
            for (int32_t d = 0; d < N; ++d) run[d] = 0;
            t = arrival_ms[next];
        }
        /* 2. FIFO admission */
        for (int32_t d = 0; d < N; ++d) {
            while (nfifo[d] > 0 && K[d] + DEMAND(fifo[(size_t)d * n]) <= C) {
                int64_t i = fifo[(size_t)d * n];
                for (int64_t k = 1; k < nfifo[d]; ++k) fifo[(size_t)d * n + k - 1] = fifo[(size_t)d * n + k];
                nfifo[d] -= 1;
                if (policy == 1 && bound[i] >= 0) R[d] -= NEED(i);
                K[d] += DEMAND(i);
                ready[(size_t)d * n + nready[d]++] = i;
            }
        }
        /* 3. arrivals at t */
        while (next < n && arrival_ms[next] == t) {
            int64_t i = next++;
            int32_t d;
            if (policy == 1 && bound[i] >= 0) {
                int32_t feas = -1, most = 0;
                for (int32_t k = 0; k < N; ++k) {
                    int64_t beff = C - K[k] - R[k];
                    if (NEED(i) <= beff && (feas < 0 || nfifo[k] < nfifo[feas])) feas = k;
                    if (beff > C - K[most] - R[most]) most = k;
                }
                d = feas >= 0 ? feas : most;
            } else {
                d = (int32_t)(i % N);
            }
            routed[i] = d;
            if (nfifo[d] == 0 && K[d] + DEMAND(i) <= C) {
                K[d] += DEMAND(i);
                ready[(size_t)d * n + nready[d]++] = i;
            } else {
                fifo[(size_t)d * n + nfifo[d]++] = i;
                if (policy == 1 && bound[i] >= 0) R[d] += NEED(i);
            }
        }
        /* 4. the state over [t, t+1) */
        for (int32_t d = 0; d < N; ++d) {
            if (K[d] * 1000000 >= (int64_t)theta_ppm * C) {
                if (run[d] == 0) hp_count[d] += 1;
                run[d] += 1;
                hp_time[d] += 1;
                hp_max[d] = max64(hp_max[d], run[d]);
            } else {
                run[d] = 0;
            }
            queue_area[d] += nfifo[d];
            max_queue[d] = max64(max_queue[d], nfifo[d]);
        }
        /* 5. one token per decoder, for the head of its ready queue */
        for (int32_t d = 0; d < N; ++d) {
            if (nready[d] == 0) continue;
            int64_t* rq = ready + (size_t)d * n;
            int64_t i = rq[0];
            for (int64_t k = 1; k < nready[d]; ++k) rq[k - 1] = rq[k];
            nready[d] -= 1;
            left[i] -= 1;
            if (left[i] == 0) release[d] = i;
            else rq[nready[d]++] = i;
        }
        t += 1;
    }
#undef DEMAND
#undef NEED
    free(ready); free(fifo); free(nready); free(nfifo); free(K); free(R); free(release); free(run); free(left);
    return 0;
}
