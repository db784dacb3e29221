// KV pressure of decoders under round-robin or MAPS routing (App. A) on
// gfx950: a batch of independent simulations, one wavefront each.
//
// Each simulation follows the requests of one arrival sequence through N
// decoders of C KV tokens (App. A: demand M = L_p + L_out held from admission
// to completion, FIFO admission while K + M <= C, one token per millisecond
// per decoder shared by its admitted requests in one-token time slices) and
// records the high-pressure intervals (K / C >= theta) of every decoder.
//
// The state only changes at arrivals and completions, so the wavefront jumps
// from one such event to the next instead of stepping through milliseconds.
// A decoder's ready queue is kept in LDS in service order (ids and tokens
// left); between events it is brought up to date lazily: after m one-token
// slices over n requests, the request at position k has received
// m / n + [k < m mod n] tokens and the queue has rotated by m mod n (the lanes
// read every entry, then write it back rotated).  The request at position k
// completes after (left_k - 1) n + k + 1 slices, so the decoder's next
// completion is a wavefront minimum; it stays valid until the decoder's queue
// changes.  When a completion is due the completing request is the last of
// the rotated queue, and an admission appends at the end: both O(1).  The
// ready queue keeps each request's demand beside it, and the next 64
// arrivals (time, prompt, output, bound) sit in the lanes' registers, so
// neither a completion nor an arrival waits on a global load.  The FIFO
// queues live in the workspace (one ring per decoder, 16 bytes an entry:
// id, prompt, output, bound), the head's entry and the per-decoder counters
// in LDS, so only an admission from a queue loads (its successor's entry).  Every loop is bounded: an arrival or a completion is
// consumed per event, and a simulation that could not progress reports an
// error instead of spinning.
#include "maps_internal.hpp"

namespace maps {
namespace {

constexpr int kSimNT = kWave;      // one wavefront per simulation
constexpr int kMaxDec = MAPS_MAX_SIM_DECODERS;
static_assert(kMaxDec <= kWave, "each decoder's state lives in one lane");
constexpr int kReady = MAPS_MAX_SIM_READY;
constexpr int kPerLane = kReady / kWave;
constexpr int64_t kNever = INT64_MAX;

struct SimArgs {
    int32_t N;
    int64_t C;
    int32_t theta_ppm;
    int64_t n;
    int32_t S;
    const int64_t* arrival;   // [S][n]
    const int32_t* prompt;    // [n]
    const int32_t* output;    // [n]
    const int32_t* bound;     // [n]
    const int32_t* policy;    // [S]
    int64_t* finish;          // [S][n]
    int32_t* routed;          // [S][n] (nullable)
    int64_t* stats;           // [S][5][N]: hp_time, hp_max, hp_count, max_queue, queue_area
    int64_t* span;            // [S][2]
    int4* fifo;               // workspace [S][N][n]: {id, prompt, output, bound}
    uint32_t* dev_err;
};

// Decoder d's state lives in lane d's registers (N <= 8 < 64): every lane
// reads it with readlane at the uniform index d, lane d alone writes it.
struct DecRegs {
    int64_t K, R;             // tokens held; needs reserved by queued requests (policy 1)
    int64_t next_done;        // time of the next completion (kNever when the ready queue is empty)
    int64_t t_sync;           // the ready queue's tokens-left are as of this time
    int64_t run, hp_time, hp_max, hp_count, max_queue, queue_area;
    int32_t nready, q_head, q_count;
    int4 head;                // the FIFO head's {id, prompt, output, bound} while q_count > 0
};

__device__ inline int32_t rl32(int32_t v, int j) { return __builtin_amdgcn_readlane(v, j); }
__device__ inline int64_t rl64(int64_t v, int j) {
    return int64_t((uint64_t(uint32_t(__builtin_amdgcn_readlane(int32_t(uint64_t(v) >> 32), j))) << 32) |
                   uint32_t(__builtin_amdgcn_readlane(int32_t(v), j)));
}

__global__ __launch_bounds__(kSimNT) void simulate_kernel(SimArgs a) {
    extern __shared__ int32_t lds[];
    const int s = blockIdx.x;
    const int lane = threadIdx.x;
    const int32_t N = a.N;
    const int64_t n = a.n, C = a.C;
    int32_t* rid = lds;                         // [N][kReady] request ids in service order
    int32_t* rleft = lds + N * kReady;          // [N][kReady] tokens left as of t_sync
    uint32_t* rdem = reinterpret_cast<uint32_t*>(lds + 2 * N * kReady);   // [N][kReady] demands L_p + L_out
    const int64_t* arr = a.arrival + int64_t(s) * n;
    int64_t* fin = a.finish + int64_t(s) * n;
    int32_t* rout = a.routed ? a.routed + int64_t(s) * n : nullptr;
    int4* fifo = a.fifo + int64_t(s) * N * n;
    const int32_t policy = a.policy[s];
    bool bad_input = false, ready_full = false;

    // The next 64 arrivals in lane registers (lane k: request wbase + k), refilled by one coalesced load
    // when the arrivals pass them; read with readlane at a uniform index.
    int64_t wbase = 0, w_arr = kNever;
    int32_t w_p = 0, w_o = 0, w_b = -1;
    auto refill = [&](int64_t base) {
        wbase = base;
        const int64_t i = base + lane;
        w_arr = i < n ? arr[i] : kNever;
        w_p = i < n ? a.prompt[i] : 0;
        w_o = i < n ? a.output[i] : 0;
        w_b = i < n ? a.bound[i] : -1;
    };
    // arrival time of request `next` (kNever past the last), the window moved up to it when passed
    auto arrival_of_next = [&](int64_t nx) -> int64_t {
        if (nx >= n) return kNever;
        if (nx >= wbase + kWave) refill(nx);
        return rl64(w_arr, int(nx - wbase));
    };
    refill(0);

    DecRegs me{};   // this lane's decoder (lanes < N)
    me.next_done = kNever;
    me.t_sync = rl64(w_arr, 0);   // the first arrival

    // bring decoder d's ready queue to time t: m slices since t_sync
    auto sync = [&](int d, int64_t t) {
        const int32_t nr = rl32(me.nready, d);
        const int64_t m = t - rl64(me.t_sync, d);
        if (nr > 0 && m > 0) {
            const int64_t q = m / nr;
            const int32_t r = int32_t(m % nr);
            int32_t id[kPerLane], lf[kPerLane];
            uint32_t dm[kPerLane];
#pragma unroll
            for (int j = 0; j < kPerLane; ++j) {   // new position k takes old position (k + r) mod nr
                if (j * kWave >= nr) break;         // uniform: only the rows of 64 that hold entries
                const int32_t k = lane + j * kWave;
                if (k < nr) {
                    int32_t src = k + r;
                    src = src >= nr ? src - nr : src;
                    id[j] = rid[d * kReady + src];
                    lf[j] = int32_t(rleft[d * kReady + src] - q - (src < r ? 1 : 0));
                    dm[j] = rdem[d * kReady + src];
                }
            }
            __syncthreads();
#pragma unroll
            for (int j = 0; j < kPerLane; ++j) {
                if (j * kWave >= nr) break;
                const int32_t k = lane + j * kWave;
                if (k < nr) {
                    rid[d * kReady + k] = id[j];
                    rleft[d * kReady + k] = lf[j];
                    rdem[d * kReady + k] = dm[j];
                }
            }
            __syncthreads();
        }
        if (lane == d) me.t_sync = t;
    };
    // decoder d's next completion after a change of its ready queue (synced to t)
    auto schedule = [&](int d, int64_t t) {
        const int32_t nr = rl32(me.nready, d);
        int64_t best = kNever;
        for (int j = 0; j < kPerLane; ++j) {
            if (j * kWave >= nr) break;
            const int32_t k = lane + j * kWave;
            if (k < nr) {
                const int64_t sk = int64_t(rleft[d * kReady + k] - 1) * nr + k + 1;
                best = sk < best ? sk : best;
            }
        }
        best = -wave_reduce_max(-best);   // the wavefront minimum (kNever = INT64_MAX negates safely)
        if (lane == d) me.next_done = nr > 0 ? t + best : kNever;
    };
    // append request i (output o, demand dem) to the ready queue (synced to t)
    auto admit = [&](int d, int64_t i, int32_t o, int64_t dem, int64_t t) {
        if (rl32(me.nready, d) >= kReady) { ready_full = true; return false; }
        sync(d, t);
        const int32_t k = rl32(me.nready, d);
        if (lane == 0) {
            rid[d * kReady + k] = int32_t(i);
            rleft[d * kReady + k] = o;
            rdem[d * kReady + k] = uint32_t(dem);
        }
        if (lane == d) {
            me.nready = k + 1;
            me.K += dem;
        }
        __syncthreads();
        return true;
    };

    int64_t t = arrival_of_next(0), next = 0, done = 0, last = t;
    uint32_t dirty = 0;   // decoders whose ready queue changed at t (bit d)
    const int64_t max_events = 2 * n + 8;
    for (int64_t ev = 0;; ++ev) {
        if (ev > max_events) { bad_input = true; break; }
        // 1. completions at t: the completing request is the last of the synced queue
        for (int d = 0; d < N; ++d) {
            if (rl64(me.next_done, d) != t) continue;
            sync(d, t);
            const int32_t k = rl32(me.nready, d) - 1;
            const int64_t i = rid[d * kReady + k];
            const int64_t dem = int64_t(rdem[d * kReady + k]);
            if (lane == d) {
                me.nready = k;
                me.K -= dem;
            }
            if (lane == 0) fin[i] = t;
            done += 1;
            last = t;
            dirty |= 1u << d;
        }
        if (done >= n) break;
        // 2. FIFO admission
        for (int d = 0; d < N; ++d) {
            while (rl32(me.q_count, d) > 0) {
                const int4 h = make_int4(rl32(me.head.x, d), rl32(me.head.y, d), rl32(me.head.z, d),
                                         rl32(me.head.w, d));
                const int64_t dem = int64_t(h.y) + h.z;
                if (rl64(me.K, d) + dem > C) break;
                if (!admit(d, h.x, h.z, dem, t)) break;
                const int32_t qh = rl32(me.q_head, d), qc = rl32(me.q_count, d) - 1;
                const int32_t nh = qh + 1 == n ? 0 : qh + 1;
                if (lane == d) {
                    me.q_head = nh;
                    me.q_count = qc;
                    if (policy == 1 && h.w >= 0) me.R -= int64_t(h.y) + h.w;
                    // the next head's entry: one 16-byte load, only after an admission (lane d wrote it)
                    if (qc > 0) me.head = fifo[int64_t(d) * n + nh];
                }
                dirty |= 1u << d;
            }
        }
        // 3. arrivals at t, in index order
        while (next < n) {
            const int64_t ai = arrival_of_next(next);
            if (ai > t) break;
            const int j = int(next - wbase);
            const int32_t pi = rl32(w_p, j), oi = rl32(w_o, j), bi = rl32(w_b, j);
            const int64_t i = next++;
            const int64_t dem = int64_t(pi) + oi, nd = int64_t(pi) + bi;
            if (ai < t || pi < 0 || oi < 1 || dem > C) {
                bad_input = true;   // out of order or never admissible: dropped
                if (lane == 0) fin[i] = t;
                done += 1;
                continue;
            }
            int d;
            if (policy == 1 && bi >= 0) {   // Algorithm 1 at block size 1
                int feas = -1, most = 0;
                int32_t fq = 0;
                int64_t most_beff = 0;
                for (int k = 0; k < N; ++k) {
                    const int64_t beff = C - rl64(me.K, k) - rl64(me.R, k);
                    const int32_t qk = rl32(me.q_count, k);
                    if (nd <= beff && (feas < 0 || qk < fq)) {
                        feas = k;
                        fq = qk;
                    }
                    if (k == 0 || beff > most_beff) {
                        most = k;
                        most_beff = beff;
                    }
                }
                d = feas >= 0 ? feas : most;
            } else {
                d = int(i % N);
            }
            if (lane == 0 && rout) rout[i] = d;
            bool queued = true;
            if (rl32(me.q_count, d) == 0 && rl64(me.K, d) + dem <= C) {
                queued = !admit(d, i, oi, dem, t);
                if (!queued) dirty |= 1u << d;
            }
            if (queued) {
                const int32_t qh = rl32(me.q_head, d), qc = rl32(me.q_count, d);
                int64_t tail = int64_t(qh) + qc;
                tail = tail >= n ? tail - n : tail;
                const int4 e = make_int4(int32_t(i), pi, oi, bi);
                if (lane == d) {   // the lane that reads the ring writes it
                    fifo[int64_t(d) * n + tail] = e;
                    if (qc == 0) me.head = e;
                    me.q_count = qc + 1;
                    if (policy == 1 && bi >= 0) me.R += nd;
                }
            }
        }
        if (done >= n) break;   // only dropped requests were left
        for (int d = 0; d < N; ++d)
            if (dirty & (1u << d)) schedule(d, t);
        dirty = 0;
        // the next event, and the state recorded over [t, t_next)
        int64_t t_next = arrival_of_next(next);
        for (int d = 0; d < N; ++d) {
            const int64_t nd = rl64(me.next_done, d);
            t_next = nd < t_next ? nd : t_next;
        }
        if (t_next == kNever || t_next <= t) { bad_input = true; break; }
        const int64_t len = t_next - t;
        if (lane < N) {
            if (me.K * 1000000 >= int64_t(a.theta_ppm) * C) {
                if (me.run == 0) me.hp_count += 1;
                me.run += len;
                me.hp_time += len;
                me.hp_max = me.run > me.hp_max ? me.run : me.hp_max;
            } else {
                me.run = 0;
            }
            me.queue_area += int64_t(me.q_count) * len;
            me.max_queue = me.q_count > me.max_queue ? me.q_count : me.max_queue;
        }
        t = t_next;
    }
    if (lane < N) {
        int64_t* o = a.stats + int64_t(s) * 5 * N;
        o[0 * N + lane] = me.hp_time;
        o[1 * N + lane] = me.hp_max;
        o[2 * N + lane] = me.hp_count;
        o[3 * N + lane] = me.max_queue;
        o[4 * N + lane] = me.queue_area;
    }
    if (lane == 0) {
        a.span[2 * int64_t(s)] = arr[0];
        a.span[2 * int64_t(s) + 1] = last;
        if (bad_input) raise_error(a.dev_err, MAPS_ERR_SIM_INPUT);
        if (ready_full) raise_error(a.dev_err, MAPS_ERR_SIM_READY);
    }
}

}  // namespace
}  // namespace maps

using namespace maps;

extern "C" size_t maps_simulate_workspace_size(int32_t N, int64_t n, int32_t S) {
    if (N < 1 || N > MAPS_MAX_SIM_DECODERS || n < 1 || S < 0) return 0;
    return align256(size_t(S) * size_t(N) * size_t(n) * sizeof(int4));
}

extern "C" maps_status maps_simulate(int32_t N, int64_t C, int32_t theta_ppm, int64_t n, int32_t S,
                                     const int64_t* arrival_ms, const int32_t* prompt, const int32_t* output,
                                     const int32_t* bound, const int32_t* policy, int64_t* finish_ms,
                                     int32_t* routed, int64_t* stats, int64_t* span, uint32_t* dev_err,
                                     void* workspace, size_t workspace_bytes, hipStream_t stream) {
    if (N < 1 || N > MAPS_MAX_SIM_DECODERS || C < 1 || n < 1 || n > INT32_MAX || S < 0 || theta_ppm < 1 ||
        theta_ppm > 1000000)
        return MAPS_E_SIZE;
    if (S == 0) return MAPS_OK;
    if (!arrival_ms || !prompt || !output || !bound || !policy || !finish_ms || !stats || !span || !dev_err ||
        !workspace)
        return MAPS_E_NULL;
    if (workspace_bytes < maps_simulate_workspace_size(N, n, S)) return MAPS_E_WORKSPACE;
    SimArgs a{N, C, theta_ppm, n, S, arrival_ms, prompt, output, bound, policy, finish_ms, routed, stats, span,
              static_cast<int4*>(workspace), dev_err};
    const size_t lds = size_t(N) * kReady * 3 * sizeof(int32_t);
    allow_dynamic_lds(simulate_kernel, lds);
    hipLaunchKernelGGL(simulate_kernel, dim3(unsigned(S)), dim3(kSimNT), lds, stream, a);
    MAPS_CHECK_LAUNCH();
    return MAPS_OK;
}
