/*
 * maps.h -- C ABI of the MAPS scheduler core for AMD Instinct MI355X (gfx950).
 *
 * MAPS (Memory-Aware Predictive Scheduling) turns speculative output-length
 * predictions into calibrated upper bounds, projects each decoder's future
 * KV-cache occupancy from its resident requests, places arriving requests on
 * decoders, and orders each decoder's local queue.  This library computes
 * those four steps for whole batches on one GPU.
 *
 * Conventions shared by every entry point
 *   - Array arguments are DEVICE pointers unless the comment says otherwise.
 *     All arrays are dense, C-contiguous and owned by the caller; the library
 *     keeps no pointer after a call returns.
 *   - Lengths are int32 token counts (one KV-cache block per token: block
 *     size S = 1).  Offsets of decoder-major segments are int64.
 *   - Work is enqueued on `stream` (NULL = the null stream) and completes
 *     asynchronously; outputs are valid once the stream is synchronized.
 *   - The library never allocates or frees device memory.  Scratch memory is
 *     the caller's `workspace` of at least the matching *_workspace_size()
 *     bytes (any alignment of 256 bytes or more; NULL is allowed when the size
 *     is 0).  A workspace may be reused once the call that used it finished.
 *   - Argument errors detectable on the host are returned synchronously as a
 *     negative maps_status and nothing is enqueued.  Errors in the VALUES of
 *     device arrays are reported by OR-ing MAPS_ERR_* bits into the device
 *     word *dev_err (never cleared by the library; the caller zeroes it).  When
 *     a bit is set the outputs of that call are unspecified, but every kernel
 *     still stays within the bounds of the buffers it was given.
 *   - Results are deterministic: the same inputs give bit-identical outputs.
 *   - Calls on different streams may run concurrently if they share no
 *     output, snapshot or workspace buffer.
 */
#ifndef MAPS_H
#define MAPS_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t maps_status;

enum {
    MAPS_OK = 0,
    MAPS_E_NULL = -1,        /* a required pointer is NULL */
    MAPS_E_SIZE = -2,        /* a count or size is out of range */
    MAPS_E_ALPHA = -3,       /* alpha_ppm is not in (0, 1000000) */
    MAPS_E_WORKSPACE = -4,   /* workspace smaller than the size query */
    MAPS_E_HIP = -5,         /* a HIP runtime call or kernel launch failed */
    MAPS_E_POLICY = -6,      /* unknown placement policy */
    MAPS_E_BUFFER = -7       /* snapshot buffer smaller than maps_snapshot_bytes() */
};

/* Quantile of a bucket whose conformal rank exceeds its size (infinite). */
#define MAPS_Q_INF INT32_MAX

/* Bits OR-ed into *dev_err. */
enum {
    MAPS_ERR_NEG_LEN = 1u,          /* a length, capacity or queue length < 0 where
                                       one is required */
    MAPS_ERR_EDGES_UNSORTED = 2u,   /* bucket edges not non-decreasing */
    MAPS_ERR_INT32_RANGE = 4u,      /* a projected occupancy could exceed INT32_MAX */
    MAPS_ERR_SEG_OFFSETS = 8u,      /* segment offsets not non-decreasing in [0, total] */
    MAPS_ERR_BOUND_RANGE = 16u,     /* a remaining length max(U-g,0) exceeds u_max */
    MAPS_ERR_SNAPSHOT = 32u,        /* snapshot was not built for this (D, u_max) */
    MAPS_ERR_QUEUE_TOO_LONG = 64u,  /* a local queue longer than MAPS_MAX_LOCAL_QUEUE */
    MAPS_ERR_TOO_MANY = 128u,       /* a decoder with MAPS_MAX_RESIDENTS or more residents */
    MAPS_ERR_WAIT_TIMEOUT = 256u,   /* reserved: no entry point raises it any more (a
                                       bounded wait on another workgroup now falls back
                                       to computing the value itself) */
    MAPS_ERR_SEEN_RANGE = 512u,     /* a seen count outside [0, n] (sliding-window
                                       calibration) */
    MAPS_ERR_BLOCK_RANGE = 1024u,   /* an effective block count left (-2^52, 2^52)
                                       during reserving placement */
    MAPS_ERR_SIM_INPUT = 2048u,     /* simulation: a request with L_p < 0, L_out < 1 or
                                       L_p + L_out > C, or arrival times that decrease
                                       (such a request is dropped) */
    MAPS_ERR_SIM_READY = 4096u      /* simulation: a decoder would have held more than
                                       MAPS_MAX_SIM_READY admitted requests */
};

/* Largest u_max (cap on bounds and remaining lengths) the snapshot accepts,
 * and the resident count per decoder it supports: 24-bit operands. */
#define MAPS_MAX_U_MAX ((1 << 24) - 64)
#define MAPS_MAX_RESIDENTS ((1 << 24) - 1)

/* Longest pending queue of one decoder that maps_local_order accepts. */
#define MAPS_MAX_LOCAL_QUEUE 2048

/* Longest calibration window and most length buckets that
 * maps_calibrate_window accepts. */
#define MAPS_MAX_WINDOW 4096
#define MAPS_MAX_WINDOW_BUCKETS 1024

/* Most decoders that maps_place_static accepts with reservation. */
#define MAPS_MAX_RESERVE_DECODERS 1024

/* Most decoders and largest u_max of placement with sequential commit. */
#define MAPS_MAX_COMMIT_DECODERS 8192
#define MAPS_MAX_COMMIT_U_MAX (1 << 20)

/* Most decoders of one simulation and most admitted requests per decoder. */
#define MAPS_MAX_SIM_DECODERS 8
#define MAPS_MAX_SIM_READY 1024

/* Largest u_max and block size of the placement in blocks. */
#define MAPS_MAX_BLOCKS_U_MAX 131072
#define MAPS_MAX_BLOCK_SIZE 64

/* Placement policies: minimum queue among feasible decoders with the largest
 * slack as fallback (Sec. 3.3 and Algorithm 1), or largest slack alone (the
 * maximum-capacity ablation of Sec. 4). */
enum { MAPS_POLICY_MQ = 0, MAPS_POLICY_MC = 1 };

/* ------------------------------------------------------------------------ */
/* 0. Capacities in bytes (App. A: KV tokens and bytes are related by model  */
/*    constants)                                                             */
/* ------------------------------------------------------------------------ */
/*
 * capacity_tokens[d] = floor(capacity_bytes[d] / bytes_per_token) for the D
 * decoders (device arrays; int64 in, int32 out), the token capacities the
 * other calls take.  dev_err bits: NEG_LEN (a negative byte count: 0 tokens),
 * INT32_RANGE (more than INT32_MAX tokens: clamped).
 * Host errors: NULL, SIZE (D < 1, bytes_per_token < 1), HIP.
 */
maps_status maps_capacity_tokens(const int64_t* capacity_bytes, int32_t D, int64_t bytes_per_token,
                                 int32_t* capacity_tokens, uint32_t* dev_err, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* 1. Uncertainty-aware calibration (Sec. 3.2, Eqs. (2)-(4))                */
/* ------------------------------------------------------------------------ */
/*
 * Calibration set of n completed requests: pred[i] (prediction L_hat) and
 * truth[i] (observed output length L), both >= 0.  Request i belongs to length
 * bucket b(i) = #{j : edges[j] <= pred[i]}, edges[0..nb-2] non-decreasing.
 * Per bucket b with n_b members, scores s_i = max(0, truth - pred) (Eq. (2)):
 *   k_b = ceil((1 - alpha)(n_b + 1)),  alpha = alpha_ppm / 10^6  (exact integer)
 *   q_out[b] = the k_b-th smallest score of the bucket (1-indexed; Eq. (3)),
 *              or MAPS_Q_INF when k_b > n_b;  count_out[b] = n_b.
 * Then, for m predictions apply_pred[0..m-1] (m may be 0; apply_pred and
 * U_out may then be NULL), the bound of Eq. (4) in the prediction's bucket:
 *   U_out[i] = -1                          if apply_pred[i] < 0 (no prediction)
 *            = u_max                       if q of its bucket is MAPS_Q_INF
 *            = min(apply_pred[i] + q, u_max) otherwise.
 * dev_err bits: NEG_LEN (pred or truth < 0), EDGES_UNSORTED.  (The bounds
 * may be written by workgroups of the selection's own launch; such a workgroup
 * waits a bounded time for each quantile and otherwise selects it itself, so
 * the call neither needs its workgroups to run at the same time nor raises
 * WAIT_TIMEOUT.)
 * Host errors: NULL, SIZE (n < 0, m < 0, nb < 1 or nb > 65536, u_max < 0),
 * ALPHA, WORKSPACE, HIP.
 */
size_t maps_calibrate_workspace_size(int64_t n, int32_t nb);
maps_status maps_calibrate(const int32_t* pred, const int32_t* truth, int64_t n,
                           const int32_t* edges, int32_t nb, int32_t alpha_ppm,
                           int32_t* q_out, int32_t* count_out,
                           const int32_t* apply_pred, int64_t m, int32_t u_max, int32_t* U_out,
                           uint32_t* dev_err, void* workspace, size_t workspace_bytes,
                           hipStream_t stream);

/*
 * maps_calibrate for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same arguments, outputs and errors without the workspace.  Its scratch
 * is a library-owned device array of MAPS_CALIBRATE_NOALLOC_BYTES per GPU
 * (held until the process ends), enough for n <= 1,048,576 residuals and
 * nb <= 1,024 buckets; a call needing more returns MAPS_E_SIZE.  The call
 * allocates nothing.  Every call on one GPU shares that array, so calls that
 * overlap on one GPU (different streams, or host threads) race: serialize
 * them on one stream.
 */
#define MAPS_CALIBRATE_NOALLOC_BYTES (8u << 20)
maps_status maps_calibrate_noalloc(const int32_t* pred, const int32_t* truth, int64_t n,
                                   const int32_t* edges, int32_t nb, int32_t alpha_ppm,
                                   int32_t* q_out, int32_t* count_out,
                                   const int32_t* apply_pred, int64_t m, int32_t u_max, int32_t* U_out,
                                   uint32_t* dev_err, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* 1b. Sliding-window calibration (Sec. 3.2: the calibration set holds the  */
/*     most recent completed requests; Sec. 4: a window of the last 500)    */
/* ------------------------------------------------------------------------ */
/*
 * Completion log of n requests, oldest first: pred[i], truth[i] >= 0, bucket
 * b(i) = #{j : edges[j] <= pred[i]} as for maps_calibrate (edges[0..nb-2]
 * non-decreasing).  Request j (0 <= j < m) with prediction apply_pred[j] had
 * seen the first apply_seen[j] log entries (0 <= apply_seen[j] <= n) when its
 * bound was taken.  Its calibration set is the `window` most recent of those
 * entries in its bucket (all of them when the bucket had fewer): n_w scores
 * s = max(0, truth - pred) (Eq. (2)), k = ceil((1 - alpha)(n_w + 1)), and
 *   q_out[j] = the k-th smallest of them (Eq. (3)), MAPS_Q_INF when k > n_w
 *              (an empty set included), -1 when apply_pred[j] < 0;
 *   U_out[j] = -1 when apply_pred[j] < 0, u_max when q is MAPS_Q_INF, else
 *              min(apply_pred[j] + q, u_max) (Eq. (4)).
 * With window >= n and every apply_seen[j] = n this is maps_calibrate's
 * bound.  All arrays are device arrays; q_out may be NULL; apply_seen is
 * int64.  m may be 0 (nothing is enqueued).
 * dev_err bits: NEG_LEN (pred or truth < 0 in the log), EDGES_UNSORTED,
 * SEEN_RANGE.  Outputs are unspecified when *dev_err != 0 (the kernels stay
 * inside their buffers).
 * Host errors: NULL, SIZE (n < 0 or n > INT32_MAX, m < 0, nb < 1 or nb >
 * MAPS_MAX_WINDOW_BUCKETS, window < 1 or window > MAPS_MAX_WINDOW,
 * u_max < 0), ALPHA, WORKSPACE (smaller than
 * maps_calibrate_window_workspace_size(n, nb)), HIP.
 */
size_t maps_calibrate_window_workspace_size(int64_t n, int32_t nb);
maps_status maps_calibrate_window(const int32_t* pred, const int32_t* truth, int64_t n,
                                  const int32_t* edges, int32_t nb, int32_t window, int32_t alpha_ppm,
                                  const int32_t* apply_pred, const int64_t* apply_seen, int64_t m,
                                  int32_t u_max, int32_t* q_out, int32_t* U_out,
                                  uint32_t* dev_err, void* workspace, size_t workspace_bytes,
                                  hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* 1c. Incremental sliding-window calibration (Sec. 3.2: the calibration    */
/*     set holds the most recent completed requests; Sec. 4: window 500)    */
/* ------------------------------------------------------------------------ */
/*
 * A caller-owned device state of maps_window_state_bytes(nb, window) bytes
 * keeps, per length bucket b (b(i) = #{j : edges[j] <= pred[i]}, as for
 * maps_calibrate), the number of completions appended so far and the scores
 * s = max(0, truth - pred) (Eq. (2)) of its last `window` ones.
 *   maps_window_reset   empties the state (enqueued on stream).
 *   maps_window_append  appends k completions (pred[k], truth[k] >= 0, in
 *                       completion order) to the log: only the newest `window`
 *                       entries of each bucket are written, the rest of the
 *                       state is untouched.  workspace of
 *                       maps_window_append_workspace_size(k, nb) bytes.
 *   maps_window_bounds  for the log as it stands (n entries appended in all):
 *                       q_out[b] = the k-th smallest of bucket b's last
 *                       n_w = min(count_b, window) scores, k = ceil((1 -
 *                       alpha)(n_w + 1)) (Eq. (3)), MAPS_Q_INF when k > n_w;
 *                       and for m predictions U_out[j] = -1 (apply_pred < 0),
 *                       u_max (infinite q) or min(apply_pred + q, u_max)
 *                       (Eq. (4)).  This is maps_calibrate_window with every
 *                       apply_seen = n.
 * dev_err bits: NEG_LEN, EDGES_UNSORTED (append); SNAPSHOT when the state was
 * not reset for these (nb, window).
 * Host errors: NULL, SIZE (nb < 1 or nb > MAPS_MAX_WINDOW_BUCKETS, window < 1
 * or window > MAPS_MAX_WINDOW, k < 0 or k > INT32_MAX, m < 0, u_max < 0),
 * ALPHA, BUFFER (state smaller than maps_window_state_bytes), WORKSPACE, HIP.
 */
size_t maps_window_state_bytes(int32_t nb, int32_t window);
size_t maps_window_append_workspace_size(int64_t k, int32_t nb);
maps_status maps_window_reset(void* state, size_t state_bytes, int32_t nb, int32_t window, hipStream_t stream);
maps_status maps_window_append(void* state, size_t state_bytes, int32_t nb, int32_t window,
                               const int32_t* pred, const int32_t* truth, int64_t k, const int32_t* edges,
                               uint32_t* dev_err, void* workspace, size_t workspace_bytes, hipStream_t stream);
maps_status maps_window_bounds(const void* state, size_t state_bytes, int32_t nb, int32_t window,
                               int32_t alpha_ppm, const int32_t* edges, const int32_t* apply_pred, int64_t m,
                               int32_t u_max, int32_t* q_out, int32_t* U_out, uint32_t* dev_err,
                               hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* 2. Projection of KV occupancy per decoder (Sec. 3.3; App. A, Eq. (8))    */
/* ------------------------------------------------------------------------ */
/*
 * D decoders; the residents of decoder d are indices [seg_off[d], seg_off[d+1])
 * of prompt/generated/upper (n_total = seg_off[D] entries, all >= 0).  A
 * resident with prompt p, g generated tokens and bound U holds p+g+t KV tokens
 * at future decoding step t while t <= R = max(U-g, 0), then frees them.
 * The occupancy O_d(t) is the sum over residents.  The call writes
 *   base_peak[d] = max_t O_d(t)   (0 for a decoder without residents)
 * and an opaque snapshot (caller-allocated, maps_snapshot_bytes(D, n_total,
 * u_max) bytes) that maps_place and maps_local_order read; it stays valid
 * until the caller overwrites it and describes the residents at call time.
 * Requires every R <= u_max.
 * dev_err bits: NEG_LEN, SEG_OFFSETS, BOUND_RANGE, INT32_RANGE (when
 * sum_r (p+g+R) + u_max > INT32_MAX for a decoder), TOO_MANY.
 * Host errors: NULL, SIZE (D < 1, n_total < 0, u_max < 0 or u_max > MAPS_MAX_U_MAX),
 * BUFFER, WORKSPACE, HIP.
 */
size_t maps_snapshot_bytes(int32_t D, int64_t n_total, int32_t u_max);
size_t maps_project_workspace_size(int32_t D, int64_t n_total, int32_t u_max);
maps_status maps_project(int32_t D, const int64_t* seg_off, int64_t n_total,
                         const int32_t* prompt, const int32_t* generated, const int32_t* upper,
                         int32_t u_max, void* snapshot, size_t snapshot_bytes, int32_t* base_peak,
                         uint32_t* dev_err, void* workspace, size_t workspace_bytes,
                         hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* 3. Global placement (Sec. 3.3 and Algorithm 1, App. C)                   */
/* ------------------------------------------------------------------------ */
/*
 * A arriving requests a = (a_prompt[a], a_upper[a]); an arrival holds p+t KV
 * tokens at step t while t <= U.  For every decoder d (snapshot of
 * maps_project with the same D and u_max):
 *   peak(a,d) = max_t [ O_d(t) + (t <= U ? p + t : 0) ],   slack = capacity[d] - peak.
 * Decoder d is feasible for a when slack >= 0.  Choice:
 *   MAPS_POLICY_MQ: the feasible decoder with the smallest queue_len[d] (Q_k);
 *                   if none is feasible, the largest slack;
 *   MAPS_POLICY_MC: the largest slack;
 *   ties go to the lowest decoder index.  An arrival with a_upper < 0 has no
 *   bound and is routed round-robin (App. A, Eq. (9)):
 *   choice = (rr_offset + a) mod D.
 * Outputs per arrival: choice[a]; chosen_peak[a] = peak(a, choice) (-1 for
 * round-robin); chosen_overflow[a] = max(0, -slack) (0 for round-robin);
 * flags[a] bit0 = chosen decoder feasible, bit1 = routed round-robin.
 * pair_peak (optional, NULL to skip): decoder-major [D][A] int32 peak(a,d),
 * -1 for round-robin arrivals.  Arrivals are evaluated independently against
 * the same snapshot (no reservation between them).
 * workspace: device memory of maps_place_workspace_size(D, A, u_max) bytes
 * (per-group partial choices), required when A > 0; the caller owns it and
 * it must not be shared by calls in flight at the same time.
 * dev_err bits: NEG_LEN (a_prompt, capacity or queue_len < 0), INT32_RANGE
 * (an arrival whose p + U could overflow a peak), SNAPSHOT.
 * Host errors: NULL (also a NULL workspace with A > 0), SIZE (D < 1, A < 0,
 * rr_offset < 0), POLICY, WORKSPACE (workspace_bytes too small), HIP.
 */
size_t maps_place_workspace_size(int32_t D, int64_t A, int32_t u_max);
maps_status maps_place(const void* snapshot, int32_t D, int32_t u_max,
                       const int32_t* capacity, const int32_t* queue_len,
                       const int32_t* a_prompt, const int32_t* a_upper, int64_t A,
                       int32_t policy, int64_t rr_offset,
                       int32_t* choice, int32_t* chosen_peak, int32_t* chosen_overflow,
                       uint8_t* flags, int32_t* pair_peak,
                       uint32_t* dev_err, void* workspace, size_t workspace_bytes,
                       hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* 3a. Placement with sequential commit (Sec. 3.3: each dispatch atomically */
/*     reserves its demand before the next request is placed; Algorithm 1)  */
/* ------------------------------------------------------------------------ */
/*
 * maps_place's rule for arrivals a = 0..A-1 taken one after another, each
 * seeing the arrivals before it: after arrival a chooses decoder d, it is
 * committed to d -- it holds p_a + t at step t while t <= U_a, like a
 * resident with g = 0 and R = U_a -- and d's queue length grows by one.  So
 *   peak(a, d) = max_t [ O_d(t) + sum_{b < a, choice b = d} [t <= U_b](p_b + t)
 *                        + [t <= U_a](p_a + t) ],
 * and policy MQ compares the running queue lengths queue_len[d] + (arrivals
 * already sent to d).  An arrival without a bound (a_upper < 0) goes round
 * robin, (rr_offset + a) mod D, joins that queue and commits no occupancy.
 * The snapshot is maps_project's for (D, u_max); every a_upper <= u_max.
 * Outputs per arrival: choice, chosen_peak (int64, -1 for round robin),
 * chosen_overflow (int64, max(0, peak - capacity)), flags (bit0 feasible,
 * bit1 round robin); queue_out [D] (nullable): queue lengths after the batch.
 * With A = 1 the outputs equal maps_place's.
 * workspace: maps_place_commit_workspace_size(D, u_max) bytes (three dense
 * int64 arrays over the step axis and one int64 per 1,024 steps per decoder:
 * about 24 (u_max + 1) bytes per decoder), caller-owned, not shared by calls
 * in flight.  The chain is serial: one workgroup takes the arrivals in order.
 * dev_err bits: NEG_LEN (a_prompt of an arrival with a bound, capacity or
 * queue_len < 0), BOUND_RANGE (a_upper > u_max: evaluated at u_max),
 * SNAPSHOT.
 * Host errors: NULL, SIZE (D < 1 or D > MAPS_MAX_COMMIT_DECODERS, A < 0,
 * rr_offset < 0, u_max < 0 or u_max > MAPS_MAX_COMMIT_U_MAX), POLICY,
 * WORKSPACE, HIP.
 */
size_t maps_place_commit_workspace_size(int32_t D, int32_t u_max);
maps_status maps_place_commit(const void* snapshot, int32_t D, int32_t u_max, const int32_t* capacity,
                              const int32_t* queue_len, const int32_t* a_prompt, const int32_t* a_upper,
                              int64_t A, int32_t policy, int64_t rr_offset, int32_t* choice,
                              int64_t* chosen_peak, int64_t* chosen_overflow, uint8_t* flags,
                              int32_t* queue_out, uint32_t* dev_err, void* workspace,
                              size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* 3b. Algorithm 1 on block counts (Sec. 3.3: runtime state, Eq. (6),       */
/*     Algorithm 1, the atomic reservation of B_need after a dispatch)      */
/* ------------------------------------------------------------------------ */
/*
 * Runtime state of D decoders in blocks of S >= 1 tokens, from the residents
 * of maps_project (seg_off, prompt p, generated g, bound U; U < 0: no bound)
 * and capacity[d] in tokens: a resident holds ceil((p+g)/S) blocks and keeps
 * reserved the blocks still missing to its demand ceil((p+U)/S) (none when
 * U < 0 or when it holds more already);
 *   b_free[d] = floor(capacity[d] / S) - sum of held blocks,
 *   b_res[d]  = sum of reserved blocks,  b_eff[d] = b_free[d] - b_res[d].
 * Staged reservation (the appendix on the global scheduling algorithm: the
 * prompt part of a dispatch's reservation is released once the prompt KV
 * reaches the decoder): in_flight (nullable, one byte per request) marks
 * requests dispatched to the decoder whose prompt KV is still in transfer;
 * such a request holds no block and reserves its whole budget
 * ceil((p+U)/S) (ceil(p/S) without a bound); g is ignored for it.  When its
 * transfer completes the caller clears its flag with g = 0: the prompt's
 * blocks move from reserved to held and B_eff is unchanged.
 * Outputs int64 [D], device arrays.  dev_err bits: NEG_LEN (p, g or capacity
 * < 0), SEG_OFFSETS.  Host errors: NULL, SIZE (D < 1, n_total < 0, S < 1), HIP.
 */
maps_status maps_rsc_state(int32_t D, const int64_t* seg_off, int64_t n_total, const int32_t* prompt,
                           const int32_t* generated, const int32_t* upper, const uint8_t* in_flight,
                           const int32_t* capacity,
                           int32_t block_size, int64_t* b_free, int64_t* b_res, int64_t* b_eff,
                           uint32_t* dev_err, hipStream_t stream);

/*
 * Algorithm 1 for arrivals a = 0..A-1 in order against the state (b_eff[D]
 * int64, queue_len[D]): B_need = ceil((a_prompt + a_upper) / S) (Eq. (6));
 * decoders with B_need <= B_eff are feasible; policy MQ takes the feasible
 * decoder with the shortest queue (lowest index on ties), else the largest
 * B_eff (lowest index on ties); policy MC always the largest B_eff.  An
 * arrival without a bound (a_upper < 0) goes round robin, (rr_offset + a) mod D,
 * with b_need = -1.
 * reserve = 0: every arrival sees the given state (independent decisions, in
 * parallel).  reserve = 1: each dispatch reserves its B_need on its decoder
 * and joins its queue before the next arrival (B_eff -= B_need, Q += 1; a
 * round-robin dispatch only joins the queue), one arrival after another;
 * D <= MAPS_MAX_RESERVE_DECODERS.
 * Outputs [A]: choice, b_need (int64), flags (bit0: B_need <= B_eff of the
 * chosen decoder before its reservation; bit1: round robin).  b_eff_out and
 * queue_out [D] (may be NULL) receive the state after the batch.
 * dev_err bits: NEG_LEN (a_prompt < 0 with a bound), BLOCK_RANGE.
 * Host errors: NULL, SIZE (D < 1, A < 0, S < 1, rr_offset < 0, reserve with
 * D > MAPS_MAX_RESERVE_DECODERS), POLICY, HIP.
 */
maps_status maps_place_static(int32_t D, const int64_t* b_eff, const int32_t* queue_len, int32_t block_size,
                              const int32_t* a_prompt, const int32_t* a_upper, int64_t A, int32_t policy,
                              int64_t rr_offset, int32_t reserve, int32_t* choice, int64_t* b_need,
                              uint8_t* flags, int64_t* b_eff_out, int32_t* queue_out, uint32_t* dev_err,
                              hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* 3c. Projected placement in blocks (Sec. 3.3: capacity in blocks of S      */
/*     tokens; Eq. (6): a request holds ceil(tokens / S) blocks)             */
/* ------------------------------------------------------------------------ */
/*
 * maps_project and maps_place with every count in blocks of S tokens: a
 * resident (p, g, U) holds ceil((p+g+t)/S) blocks at future step t while
 * t <= R = max(U-g, 0), an arrival (p, U) ceil((p+t)/S) while t <= U, and
 *   peak(a, d) = max_t [OB_d(t) + [t <= U_a] ceil((p_a+t)/S)]  (blocks),
 * against floor(capacity[d] / S) blocks; the choice, outputs and flags are
 * those of maps_place in blocks (chosen_peak, chosen_overflow, pair_peak).
 * With S = 1 every output equals the token path's.
 * maps_project_blocks writes the decoders' block snapshot (caller buffer of
 * maps_blocks_snapshot_bytes(D, n_total, u_max, S) bytes, valid for
 * maps_place_blocks with the same seg_off, D, n_total, u_max and S) and the
 * base peaks in blocks.  maps_place_blocks writes every pair peak into
 * pair_peak[D][A] (required) and then the choices.  1 <= S <=
 * MAPS_MAX_BLOCK_SIZE, 0 <= u_max <= MAPS_MAX_BLOCKS_U_MAX.
 * dev_err bits: NEG_LEN, BOUND_RANGE, SEG_OFFSETS, INT32_RANGE (as
 * maps_project); from maps_place_blocks NEG_LEN (a_prompt of an arrival with a
 * bound, capacity or queue_len < 0), INT32_RANGE (a pair peak above INT32_MAX,
 * stored clamped), and SNAPSHOT when the snapshot was not
 * written by maps_project_blocks for these D, n_total, u_max and S, or a
 * decoder's resident count under seg_off differs from the one it was built
 * with (that call then reads no slice).  Host errors: NULL, SIZE, BUFFER,
 * POLICY, HIP.
 */
size_t maps_blocks_snapshot_bytes(int32_t D, int64_t n_total, int32_t u_max, int32_t block_size);
maps_status maps_project_blocks(int32_t D, const int64_t* seg_off, const int32_t* prompt,
                                const int32_t* generated, const int32_t* upper, int64_t n_total,
                                int32_t u_max, int32_t block_size, void* snapshot, size_t snapshot_bytes,
                                int32_t* base_peak, uint32_t* dev_err, hipStream_t stream);
maps_status maps_place_blocks(const void* snapshot, const int64_t* seg_off, int32_t D, int64_t n_total,
                              int32_t u_max, int32_t block_size, const int32_t* capacity,
                              const int32_t* queue_len, const int32_t* a_prompt, const int32_t* a_upper,
                              int64_t A, int32_t policy, int64_t rr_offset, int32_t* choice,
                              int32_t* chosen_peak, int32_t* chosen_overflow, uint8_t* flags,
                              int32_t* pair_peak, uint32_t* dev_err, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* 4. Local order and admission (Sec. 3.3, Eq. (7); App. A, Eq. (10))       */
/* ------------------------------------------------------------------------ */
/*
 * Pending queue of decoder d: indices [q_off[d], q_off[d+1]) of q_prompt,
 * q_upper and q_wait_ms (total = q_off[D] entries); q_upper < 0 means "no
 * bound" and counts as u_max.  Requests that waited at least max_wait_ms go
 * first in queue order (starvation guard); the rest follow sorted by bound,
 * equal bounds in queue order (Eq. (7)).  q_wait_ms may be NULL (no request
 * is promoted).  order[q_off[d] + i] is the queue-local index of the i-th
 * request of the new order.  admitted[d] is the largest k such that the
 * residents of the snapshot plus the first k reordered requests (each
 * starting now, holding p+t while t <= U) keep the projected peak <= capacity[d]
 * (0 when the residents alone exceed it).
 * dev_err bits: NEG_LEN, SEG_OFFSETS, QUEUE_TOO_LONG, SNAPSHOT.
 * Host errors: NULL, SIZE (D < 1, total < 0), WORKSPACE, HIP.
 */
size_t maps_local_order_workspace_size(int32_t D, int64_t total);
maps_status maps_local_order(const void* snapshot, int32_t D, int32_t u_max,
                             const int32_t* capacity, const int64_t* q_off, int64_t total,
                             const int32_t* q_prompt, const int32_t* q_upper,
                             const int32_t* q_wait_ms, int32_t max_wait_ms,
                             int32_t* order, int32_t* admitted,
                             uint32_t* dev_err, void* workspace, size_t workspace_bytes,
                             hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* 3 + 4. Placement and local order in two launches (Algorithm 1; Sec. 3.3, */
/*        Eq. (7))                                                           */
/* ------------------------------------------------------------------------ */
/*
 * Exactly maps_place followed by maps_local_order on the same snapshot, D,
 * u_max and capacity (the arguments keep their meaning, layout and ownership;
 * q_total is maps_local_order's `total`; one dev_err word and the placement
 * workspace of maps_place_workspace_size(D, A, u_max) bytes), with the same
 * outputs bit for bit.  The final selection of placement and every decoder's
 * local order share one launch, so the order costs no launch of its own and
 * runs beside the selection.  A may be 0 (then only the orders are computed).
 * dev_err bits: those of both calls.
 * Host errors: those of both calls; nothing is enqueued when either argument
 * set is rejected.
 */
maps_status maps_place_order(const void* snapshot, int32_t D, int32_t u_max,
                             const int32_t* capacity, const int32_t* queue_len,
                             const int32_t* a_prompt, const int32_t* a_upper, int64_t A,
                             int32_t policy, int64_t rr_offset,
                             int32_t* choice, int32_t* chosen_peak, int32_t* chosen_overflow,
                             uint8_t* flags, int32_t* pair_peak,
                             const int64_t* q_off, int64_t q_total,
                             const int32_t* q_prompt, const int32_t* q_upper,
                             const int32_t* q_wait_ms, int32_t max_wait_ms,
                             int32_t* order, int32_t* admitted,
                             uint32_t* dev_err, void* workspace, size_t workspace_bytes,
                             hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* 5. KV pressure under round-robin or MAPS routing (App. A)                */
/* ------------------------------------------------------------------------ */
/*
 * S independent simulations of N decoders with a KV capacity of C tokens
 * each, serving the same n requests (prompt[i] = L_p >= 0, output[i] = L_out
 * >= 1, bound[i] = calibrated bound or < 0 for none; host-side arrays are not
 * accepted: all are device arrays) at simulation s's arrival times
 * arrival_ms[s][i] (whole milliseconds, non-decreasing in i).  Request i holds
 * M = L_p + L_out tokens from its admission to its completion (Eq. (8)).
 * Routing, policy[s]: 0 round robin, d = i mod N (Eq. (9), decoders counted
 * from 0); 1 Algorithm 1 at block size 1 with B_need = L_p + bound,
 * B_eff(d) = C - K_d - (needs of the requests waiting in d's queue) and
 * Q_d = d's queue length (shortest queue among B_need <= B_eff, else the
 * largest B_eff, lowest index on ties; no bound: round robin).
 * Each millisecond t: (1) a request whose last token was decoded during
 * [t-1, t) completes at t and releases M; (2) every decoder admits the head
 * of its FIFO queue while K_d + M <= C (Eq. (10)); (3) the arrivals at t are
 * routed in index order and admitted at once when the decoder's queue is
 * empty and K_d + M <= C, else queued; (4) the state over [t, t+1) is
 * recorded: high pressure when K_d / C >= theta_ppm / 10^6; (5) every
 * decoder decodes one token for the request at the head of its ready queue
 * (t_tok = 1 ms; processor sharing by one-token time slices), which goes to
 * the back unless it is done; admissions join the back.
 * Outputs: finish_ms[s][i] (completion time), routed[s][i] (decoder;
 * nullable), stats[s][5][N] = per decoder the time under high pressure
 * within [first arrival, last completion), the longest high-pressure
 * interval, the number of intervals, the longest FIFO queue and the sum over
 * milliseconds of the FIFO queue length; span[s][2] = first arrival, last
 * completion.  The high-pressure fraction of App. A is stats[s][0][d] /
 * (span[s][1] - span[s][0]).
 * workspace: maps_simulate_workspace_size(N, n, S) bytes (the FIFO queues:
 * 16 bytes per request slot, S N n slots).
 * One wavefront per simulation; N <= MAPS_MAX_SIM_DECODERS and at most
 * MAPS_MAX_SIM_READY admitted requests per decoder at a time.
 * dev_err bits: SIM_INPUT, SIM_READY (outputs unspecified when set).
 * Host errors: NULL, SIZE (N out of range, C < 1, n < 1 or n > INT32_MAX,
 * S < 0, theta_ppm not in [1, 10^6]), WORKSPACE, HIP.
 */
size_t maps_simulate_workspace_size(int32_t N, int64_t n, int32_t S);
maps_status maps_simulate(int32_t N, int64_t C, int32_t theta_ppm, int64_t n, int32_t S,
                          const int64_t* arrival_ms, const int32_t* prompt, const int32_t* output,
                          const int32_t* bound, const int32_t* policy, int64_t* finish_ms,
                          int32_t* routed, int64_t* stats, int64_t* span, uint32_t* dev_err,
                          void* workspace, size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* 2 + 4. Projection and local order in one launch (Sec. 3.3; Eq. (7);      */
/*        App. A, Eq. (10))                                                  */
/* ------------------------------------------------------------------------ */
/*
 * Exactly maps_project followed by maps_local_order on the snapshot it
 * writes (same D and u_max; capacity, q_off, q_total, q_prompt, q_upper,
 * q_wait_ms, max_wait_ms, order and admitted as for maps_local_order), with
 * the same outputs bit for bit.  Each decoder's workgroup orders the
 * decoder's queue right after projecting it, so the order costs no launch
 * or pass of its own.  dev_err bits: those of both calls.  Host errors:
 * those of both calls; nothing is enqueued when either argument set is
 * rejected.
 */
maps_status maps_project_order(int32_t D, const int64_t* seg_off, int64_t n_total,
                               const int32_t* prompt, const int32_t* generated, const int32_t* upper,
                               int32_t u_max, void* snapshot, size_t snapshot_bytes, int32_t* base_peak,
                               const int32_t* capacity, const int64_t* q_off, int64_t q_total,
                               const int32_t* q_prompt, const int32_t* q_upper, const int32_t* q_wait_ms,
                               int32_t max_wait_ms, int32_t* order, int32_t* admitted,
                               uint32_t* dev_err, hipStream_t stream);

/* Static description of a status code (host). */
const char* maps_status_string(maps_status status);

#ifdef __cplusplus
}
#endif

#endif /* MAPS_H */
