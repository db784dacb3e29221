// Placement with sequential commit (Sec. 3.3: each dispatch atomically
// reserves its demand before the next request is placed; Algorithm 1) on
// gfx950.
//
// Arrivals are placed in order.  Each is evaluated against every decoder's
// projected occupancy, which includes the arrivals already committed to that
// decoder (a committed arrival (p, U) holds p + t at step t while t <= U), and
// is then committed to the decoder it chose.  Per decoder the dense step axis
// t = 0..T (T = u_max) is kept in the workspace:
//   O(t)   occupancy,
//   PF(u)  max_{t <= u} (O(t) + t)         (stored, see the floors below),
//   SA(u)  max_{t > u} O(t)                (0 at u = T),
// so that peak(p, U) = max(p + PF(U), SA(U)) is two reads.  Committing (p, U)
// changes O only on [0, U]; there PF and SA are derived again by workgroup
// scans.  Above U, PF(u) becomes max(PF(u), v) with v = PF(U) after the
// commit; instead of rewriting that tail, v is recorded as a floor for every
// u > U in a Fenwick tree of prefix maxima over the step axis (one per
// decoder), and a lookup takes max(PF(U), floors at U).  A floor never exceeds
// the true prefix maximum (O only grows), and the largest floor that applies
// restores every change made above the stored values, so the lookup is exact.
//
//   commit_init    one 1,024-thread workgroup per decoder: O(t) from the
//                  snapshot (the rank of t among the events, then S_e + t N_e),
//                  PF and SA by prefix and suffix scans, floors cleared.
//   commit_serial  one 1,024-thread workgroup for the whole chain: per arrival
//                  every decoder's peak (one thread per decoder: PF, SA and the
//                  floors of its Fenwick path), the choice by a workgroup
//                  argmin, then the commit on [0, U] of the chosen decoder and
//                  one Fenwick update.  Queue lengths and capacities live in
//                  LDS.  The chain is serial by definition.
#include "maps_internal.hpp"

namespace maps {
namespace {

constexpr int kCommitNT = 1024;
constexpr int kWaves = kCommitNT / kWave;
constexpr int64_t kFeasibleBias = int64_t(1) << 62;
constexpr int kBatch = 8;   // dense entries a thread loads at once in a commit

struct CommitLayout {
    int32_t D, L;          // decoders, steps per decoder (u_max + 1)
    size_t off_O, off_PF, off_SA, off_F, bytes;
};

CommitLayout commit_layout(int32_t D, int32_t u_max) {
    CommitLayout c;
    c.D = D;
    c.L = u_max + 1;
    const size_t dense = align256(size_t(D) * size_t(c.L) * sizeof(int64_t));
    c.off_O = 0;
    c.off_PF = dense;
    c.off_SA = 2 * dense;
    c.off_F = 3 * dense;
    c.bytes = c.off_F + align256(size_t(D) * size_t(c.L + 1) * sizeof(int64_t));
    return c;
}

struct CommitArgs {
    SnapLayout S;
    const void* snap;
    int64_t* O;
    int64_t* PF;
    int64_t* SA;
    int64_t* F;        // [D][L + 1] Fenwick tree of floors, positions 1..L (position u + 1 is step u)
    int32_t L;
    const int32_t* cap;
    const int32_t* qlen;
    const int32_t* ap;
    const int32_t* aU;
    int64_t A;
    int32_t policy;
    int64_t rr_offset;
    int32_t* choice;
    int64_t* chosen_peak;
    int64_t* chosen_over;
    uint8_t* flags;
    int32_t* queue_out;
    uint32_t* dev_err;
};

__device__ inline int64_t max64(int64_t a, int64_t b) { return a > b ? a : b; }

// ---------------------------------------------------------------------------
// Dense curves of every decoder from the snapshot
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kCommitNT) void commit_init(CommitArgs a) {
    __shared__ int64_t tmp[kWaves];
    const int d = blockIdx.x;
    const int32_t L = a.L;
    int64_t* O = a.O + int64_t(d) * L;
    int64_t* PF = a.PF + int64_t(d) * L;
    int64_t* SA = a.SA + int64_t(d) * L;
    int64_t* F = a.F + int64_t(d) * (L + 1);
    for (int32_t i = threadIdx.x; i <= L; i += kCommitNT) F[i] = 0;

    const SnapView V = snap_view(const_cast<void*>(a.snap), a.S);
    const SnapHeader* hs = V.hdr;
    bool ok = hs->magic == kSnapMagic && hs->D == a.S.D && hs->u_max == a.S.u_max && hs->W == a.S.W &&
              hs->P == a.S.P;
    DecHeader h{};
    if (ok) {
        h = V.dec[d];
        ok = slice_ok(h, hs->n_total, a.S);
    }
    if (!ok) {
        if (threadIdx.x == 0) raise_error(a.dev_err, MAPS_ERR_SNAPSHOT);
        for (int32_t t = threadIdx.x; t < L; t += kCommitNT) O[t] = PF[t] = SA[t] = 0;
        return;
    }
    const uint2* rank = slice_rank(V, h);
    const int2* cold = slice_cold(V, h, a.S);
    const uint32_t E = uint32_t(h.E);
    // occupancy at step t: the rank e of t among the events, then S_e + t N_e
    auto occ = [&](int32_t t) -> int64_t {
        const uint2 w = rank[t >> 5];
        uint32_t e = w.y + __popc(w.x & ((1u << (t & 31)) - 1u));
        e = e < E ? e : E;
        const int2 c = cold[e];
        return int64_t(c.x) + int64_t(t) * (c.y - 1);
    };
    const int32_t chunk = (L + kCommitNT - 1) / kCommitNT;
    const int32_t b = threadIdx.x * chunk, e = b + chunk < L ? b + chunk : L;
    int64_t mpre = 0, msuf = 0;
    for (int32_t t = b; t < e; ++t) {
        const int64_t o = occ(t);
        O[t] = o;
        mpre = max64(mpre, o + t);
        msuf = max64(msuf, o);
    }
    int64_t total;
    int64_t run = block_excl_scan<kCommitNT, true>(mpre, int64_t(0), tmp, &total);
    for (int32_t t = b; t < e; ++t) {
        run = max64(run, O[t] + t);
        PF[t] = run;
    }
    // suffix: the largest O over the chunks after this thread's
    __syncthreads();
    const int lane = threadIdx.x % kWave, wid = threadIdx.x / kWave;
    int64_t after = 0;
    {
        // reverse exclusive scan: thread i receives max over threads > i
        int64_t incl = msuf;
        // within the wavefront, from the top lane down: lane i sees lanes i..63
        for (int k = 1; k < kWave; k <<= 1) {
            const int64_t x = __shfl_down(incl, k, kWave);
            if (lane + k < kWave) incl = max64(incl, x);
        }
        if (lane == 0) tmp[wid] = incl;
        __syncthreads();
        for (int i = wid + 1; i < kWaves; ++i) after = max64(after, tmp[i]);
        const int64_t next = __shfl_down(incl, 1, kWave);
        if (lane + 1 < kWave) after = max64(after, next);
    }
    int64_t s = after;
    for (int32_t t = e - 1; t >= b; --t) {
        SA[t] = s;
        s = max64(s, O[t]);
    }
}

// ---------------------------------------------------------------------------
// The serial chain
// ---------------------------------------------------------------------------

// Largest floor that applies at step u: prefix maximum over Fenwick positions
// 1..u+1.  The positions are known up front, so the loads are independent.
constexpr int kFenwickSteps = 21;   // positions up to 2^21 > MAPS_MAX_COMMIT_U_MAX + 1
__device__ inline int64_t floor_at(const int64_t* F, int32_t u) {
    // every position of the path first (ALU only), then all loads, then the maximum:
    // the loads are in flight together instead of one round trip each
    int32_t pos[kFenwickSteps];
    int32_t i = u + 1;
#pragma unroll
    for (int k = 0; k < kFenwickSteps; ++k) {
        pos[k] = i;
        i -= i & -i;
    }
    int64_t x[kFenwickSteps];
#pragma unroll
    for (int k = 0; k < kFenwickSteps; ++k) x[k] = pos[k] > 0 ? F[pos[k]] : 0;
    int64_t m = 0;
#pragma unroll
    for (int k = 0; k < kFenwickSteps; ++k) m = max64(m, x[k]);
    return m;
}

// Workgroup argmin of (key, d), lowest d on ties; every thread gets the result.
__device__ inline void block_argmin(int64_t& key, int32_t& d, int64_t* skey, int32_t* sd) {
    for (int k = kWave / 2; k > 0; k >>= 1) {
        const int64_t ok = __shfl_xor(key, k, kWave);
        const int32_t od = __shfl_xor(d, k, kWave);
        if (ok < key || (ok == key && od < d)) { key = ok; d = od; }
    }
    const int lane = threadIdx.x % kWave, wid = threadIdx.x / kWave;
    if (lane == 0) { skey[wid] = key; sd[wid] = d; }
    __syncthreads();
    key = skey[0];
    d = sd[0];
    for (int i = 1; i < kWaves; ++i)
        if (skey[i] < key || (skey[i] == key && sd[i] < d)) { key = skey[i]; d = sd[i]; }
}

__global__ __launch_bounds__(kCommitNT) void commit_serial(CommitArgs a) {
    extern __shared__ int32_t lds[];
    int32_t* Q = lds;                  // [D] running queue lengths
    int32_t* C = lds + a.S.D;          // [D] capacities
    __shared__ int32_t tile_p[kCommitNT], tile_U[kCommitNT];   // the next kCommitNT arrivals
    __shared__ int64_t skey[kWaves], scan_tmp[kWaves];
    __shared__ int32_t sd[kWaves];
    __shared__ int64_t speak;
    const int32_t D = a.S.D, L = a.L, T = L - 1;
    bool neg = false;
    for (int32_t d = threadIdx.x; d < D; d += kCommitNT) {
        Q[d] = a.qlen[d];
        C[d] = a.cap[d];
        neg |= Q[d] < 0 || C[d] < 0;
    }
    if (neg) raise_error(a.dev_err, MAPS_ERR_NEG_LEN);
    __syncthreads();
    const int lane = threadIdx.x % kWave, wid = threadIdx.x / kWave;
    for (int64_t i = 0; i < a.A; ++i) {
        if (i % kCommitNT == 0) {   // stage the next tile of arrivals (the last barrier of the step precedes)
            const int64_t j = i + threadIdx.x;
            tile_p[threadIdx.x] = j < a.A ? a.ap[j] : 0;
            tile_U[threadIdx.x] = j < a.A ? a.aU[j] : -1;
            __syncthreads();
        }
        const int32_t p0 = tile_p[i % kCommitNT], U = tile_U[i % kCommitNT];
        if (U < 0) {   // no bound: round robin, the request only joins the queue
            if (threadIdx.x == 0) {
                const int32_t d = int32_t((a.rr_offset + i) % D);
                a.choice[i] = d;
                a.chosen_peak[i] = -1;
                a.chosen_over[i] = 0;
                a.flags[i] = 2;
                Q[d] += 1;
            }
            __syncthreads();
            continue;
        }
        if (threadIdx.x == 0) {
            if (p0 < 0) raise_error(a.dev_err, MAPS_ERR_NEG_LEN);
            if (U > T) raise_error(a.dev_err, MAPS_ERR_BOUND_RANGE);
        }
        const int64_t p = p0 < 0 ? 0 : p0;
        const int32_t Uc = U < T ? U : T;
        // every decoder's peak with this arrival, and the thread's best key
        int64_t key = INT64_MAX, peak_best = 0;
        int32_t best = INT32_MAX;
        for (int32_t d = threadIdx.x; d < D; d += kCommitNT) {
            const int64_t off = int64_t(d) * L + Uc;
            const int64_t pf = max64(a.PF[off], floor_at(a.F + int64_t(d) * (L + 1), Uc));
            const int64_t peak = max64(p + pf, a.SA[off]);
            const int64_t over = peak - C[d];
            const int64_t k = (a.policy == MAPS_POLICY_MQ && over <= 0) ? int64_t(Q[d]) - kFeasibleBias : over;
            if (k < key) { key = k; best = d; peak_best = peak; }
        }
        int64_t bkey = key;
        int32_t bd = best;
        block_argmin(bkey, bd, skey, sd);
        if (bd < 0 || bd >= D) bd = 0;   // unreachable with D >= 1; keeps every index in range
        if (best == bd && bd != INT32_MAX) speak = peak_best;   // the owner of the chosen decoder
        __syncthreads();
        const int64_t peak = speak;
        if (threadIdx.x == 0) {
            const int64_t over = peak - C[bd];
            a.choice[i] = bd;
            a.chosen_peak[i] = peak;
            a.chosen_over[i] = over > 0 ? over : 0;
            a.flags[i] = over <= 0 ? 1 : 0;
            Q[bd] += 1;
        }
        // commit (p, Uc) to decoder bd: O += p + t on [0, Uc], then PF and SA there
        int64_t* __restrict__ O = a.O + int64_t(bd) * L;
        int64_t* __restrict__ PF = a.PF + int64_t(bd) * L;
        int64_t* __restrict__ SA = a.SA + int64_t(bd) * L;
        const int32_t n = Uc + 1;
        const int32_t chunk = (n + kCommitNT - 1) / kCommitNT;
        const int32_t b = threadIdx.x * chunk, e = b + chunk < n ? b + chunk : n;
        const int64_t sa_top = SA[Uc];   // max of O beyond Uc: unchanged by the commit
        int64_t mpre = 0, msuf = 0;
        // kBatch loads in flight at a time, then their updates
        for (int32_t t0 = b; t0 < e; t0 += kBatch) {
            int64_t o[kBatch];
#pragma unroll
            for (int j = 0; j < kBatch; ++j) o[j] = t0 + j < e ? O[t0 + j] : 0;
#pragma unroll
            for (int j = 0; j < kBatch; ++j) {
                const int32_t t = t0 + j;
                if (t >= e) break;
                o[j] += p + t;
                O[t] = o[j];
                mpre = max64(mpre, o[j] + t);
                msuf = max64(msuf, o[j]);
            }
        }
        int64_t v;
        int64_t run = block_excl_scan<kCommitNT, true>(mpre, int64_t(0), scan_tmp, &v);
        // suffix maxima over the chunks after this thread's (scan of the reversed thread order)
        int64_t incl = msuf;
        for (int k = 1; k < kWave; k <<= 1) {
            const int64_t x = __shfl_down(incl, k, kWave);
            if (lane + k < kWave) incl = max64(incl, x);
        }
        __syncthreads();   // every wave has read scan_tmp
        if (lane == 0) scan_tmp[wid] = incl;
        __syncthreads();
        int64_t after = sa_top;
        for (int w = wid + 1; w < kWaves; ++w) after = max64(after, scan_tmp[w]);
        const int64_t next = __shfl_down(incl, 1, kWave);
        if (lane + 1 < kWave) after = max64(after, next);
        for (int32_t t0 = b; t0 < e; t0 += kBatch) {
            int64_t o[kBatch];
#pragma unroll
            for (int j = 0; j < kBatch; ++j) o[j] = t0 + j < e ? O[t0 + j] : 0;
#pragma unroll
            for (int j = 0; j < kBatch; ++j) {
                if (t0 + j >= e) break;
                run = max64(run, o[j] + t0 + j);
                PF[t0 + j] = run;
            }
        }
        for (int32_t t1 = e; t1 > b; t1 -= kBatch) {   // [t1 - kBatch, t1) from the top down
            int64_t o[kBatch];
#pragma unroll
            for (int j = 0; j < kBatch; ++j) o[j] = t1 - 1 - j >= b ? O[t1 - 1 - j] : 0;
#pragma unroll
            for (int j = 0; j < kBatch; ++j) {
                const int32_t t = t1 - 1 - j;
                if (t < b) break;
                if (t < Uc) SA[t] = after;
                after = max64(after, o[j]);
            }
        }
        // the new PF(Uc) = v is a floor for every step above Uc
        if (threadIdx.x < kFenwickSteps) {
            // lane k updates the k-th position of the path (no two lanes share one, so the
            // read-modify-writes run side by side); 64-bit positions: past L a position keeps
            // doubling and would wrap a 32-bit integer to a negative index
            int64_t j = int64_t(Uc) + 2;
            for (int k = 0; k < int(threadIdx.x) && j <= L; ++k) j += j & -j;
            if (j <= L) {
                int64_t* Fd = a.F + int64_t(bd) * (L + 1);
                Fd[j] = max64(Fd[j], v);
            }
        }
        __syncthreads();
    }
    if (a.queue_out)
        for (int32_t d = threadIdx.x; d < D; d += kCommitNT) a.queue_out[d] = Q[d];
}

}  // namespace
}  // namespace maps

using namespace maps;

extern "C" size_t maps_place_commit_workspace_size(int32_t D, int32_t u_max) {
    if (D < 1 || D > MAPS_MAX_COMMIT_DECODERS || u_max < 0 || u_max > MAPS_MAX_COMMIT_U_MAX) return 0;
    return commit_layout(D, u_max).bytes;
}

extern "C" maps_status maps_place_commit(const void* snapshot, int32_t D, int32_t u_max, const int32_t* capacity,
                                         const int32_t* queue_len, const int32_t* a_prompt, const int32_t* a_upper,
                                         int64_t A, int32_t policy, int64_t rr_offset, int32_t* choice,
                                         int64_t* chosen_peak, int64_t* chosen_overflow, uint8_t* flags,
                                         int32_t* queue_out, uint32_t* dev_err, void* workspace,
                                         size_t workspace_bytes, hipStream_t stream) {
    if (D < 1 || D > MAPS_MAX_COMMIT_DECODERS || A < 0 || rr_offset < 0 || u_max < 0 ||
        u_max > MAPS_MAX_COMMIT_U_MAX)
        return MAPS_E_SIZE;
    if (policy != MAPS_POLICY_MQ && policy != MAPS_POLICY_MC) return MAPS_E_POLICY;
    if (!snapshot || !capacity || !queue_len || !dev_err || !workspace ||
        (A > 0 && (!a_prompt || !a_upper || !choice || !chosen_peak || !chosen_overflow || !flags)))
        return MAPS_E_NULL;
    const CommitLayout c = commit_layout(D, u_max);
    if (workspace_bytes < c.bytes) return MAPS_E_WORKSPACE;
    char* w = static_cast<char*>(workspace);
    CommitArgs a{};
    a.S = snap_layout(D, 0, u_max);   // region offsets do not depend on the resident count
    a.snap = snapshot;
    a.O = reinterpret_cast<int64_t*>(w + c.off_O);
    a.PF = reinterpret_cast<int64_t*>(w + c.off_PF);
    a.SA = reinterpret_cast<int64_t*>(w + c.off_SA);
    a.F = reinterpret_cast<int64_t*>(w + c.off_F);
    a.L = c.L;
    a.cap = capacity;
    a.qlen = queue_len;
    a.ap = a_prompt;
    a.aU = a_upper;
    a.A = A;
    a.policy = policy;
    a.rr_offset = rr_offset;
    a.choice = choice;
    a.chosen_peak = chosen_peak;
    a.chosen_over = chosen_overflow;
    a.flags = flags;
    a.queue_out = queue_out;
    a.dev_err = dev_err;
    hipLaunchKernelGGL(commit_init, dim3(unsigned(D)), dim3(kCommitNT), 0, stream, a);
    MAPS_CHECK_LAUNCH();
    const size_t lds = size_t(2) * D * sizeof(int32_t);
    allow_dynamic_lds(commit_serial, lds);
    hipLaunchKernelGGL(commit_serial, dim3(1), dim3(kCommitNT), lds, stream, a);
    MAPS_CHECK_LAUNCH();
    return MAPS_OK;
}
