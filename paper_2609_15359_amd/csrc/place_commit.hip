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
// commit.  That tail is rewritten only up to the end of U's block of kFloorBlock
// steps; for the blocks after it v is recorded as a floor of the block
// (FB[k] = max(FB[k], v)), and a lookup takes max(PF(u), FB[block of u]).  A
// floor never exceeds the true prefix maximum (O only grows), and every change
// above the stored values is restored by the largest floor of an earlier
// block or the rewritten tail within the block, so the lookup is exact.
//
//   commit_init    one 1,024-thread workgroup per decoder: O(t) from the
//                  snapshot (the rank of t among the events, then S_e + t N_e),
//                  PF and SA by prefix and suffix scans, floors cleared.
//   commit_serial  one 512-thread workgroup for the whole chain: per arrival
//                  every decoder's peak (PF, SA and the block floor at U), the
//                  choice by a workgroup argmin, then the commit on [0, U] of
//                  the chosen decoder with its tail and block floors; a range
//                  that fits keeps its new O values in LDS for the two scans.
//                  Queue lengths and capacities live in LDS; with at most 512
//                  decoders the next arrival's lookups are issued with the
//                  commit's loads.  The chain is serial by definition.
#include "maps_internal.hpp"

namespace maps {
namespace {

constexpr int kCommitNT = 1024;            // threads of a workgroup building one decoder's curves
constexpr int kWaves = kCommitNT / kWave;
constexpr int kSerialNT = 512;             // threads of the chain's workgroup (256 VGPRs each: no spills)
constexpr int kSerialWaves = kSerialNT / kWave;
constexpr int64_t kFeasibleBias = int64_t(1) << 62;

constexpr int kFloorBlock = 1024;  // steps per floor block
constexpr int kFloorPer = 2;       // block floors a thread updates per commit: blocks up to 2 * kSerialNT
constexpr int kTailPer = kFloorBlock / kSerialNT;   // steps of a commit's own block above it per thread

struct CommitLayout {
    int32_t D, L, NB;      // decoders, steps per decoder (u_max + 1), floor blocks per decoder
    size_t off_O, off_PF, off_SA, off_F, bytes;
};

CommitLayout commit_layout(int32_t D, int32_t u_max) {
    CommitLayout c;
    c.D = D;
    c.L = u_max + 1;
    c.NB = (c.L + kFloorBlock - 1) / kFloorBlock;
    const size_t dense = align256(size_t(D) * size_t(c.L) * sizeof(int64_t));
    c.off_O = 0;
    c.off_PF = dense;
    c.off_SA = 2 * dense;
    c.off_F = 3 * dense;
    c.bytes = c.off_F + align256(size_t(D) * size_t(c.NB) * sizeof(int64_t));
    return c;
}
// the blocks after a commit's own: at most NB - 1
static_assert((MAPS_MAX_COMMIT_U_MAX + kFloorBlock) / kFloorBlock - 1 <= kFloorPer * kSerialNT,
              "block floors per thread");
static_assert(kTailPer * kSerialNT >= kFloorBlock - 1, "steps of a block above a commit per thread");

struct CommitArgs {
    SnapLayout S;
    const void* snap;
    int64_t* O;
    int64_t* PF;
    int64_t* SA;
    int64_t* F;        // [D][NB] block floors: the largest v of a commit in an earlier block
    int32_t L, NB;
    int32_t stage_cap;   // range entries the chain stages in LDS
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
    int64_t* F = a.F + int64_t(d) * a.NB;
    for (int32_t i = threadIdx.x; i < a.NB; i += kCommitNT) F[i] = 0;

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

constexpr int kBatch = 24;                  // range entries a thread loads at once

// Barrier that orders LDS traffic only: each wave waits for its own LDS
// operations, not for its global stores in flight (a full __syncthreads waits
// for those too, about a microsecond after the commit's stores).  The memory
// clobber keeps the compiler from moving memory accesses across it.
__device__ inline void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Exclusive max-scan of one value per thread over the chain's workgroup, with
// LDS-only barriers; the total goes to *total.
__device__ inline int64_t chain_excl_max(int64_t v, int64_t* tmp, int64_t* total) {
    const int lane = threadIdx.x % kWave, wid = threadIdx.x / kWave;
    const int64_t incl = wave_incl_scan_max(v);
    lds_barrier();   // every wave has read tmp's earlier contents
    if (lane == kWave - 1) tmp[wid] = incl;
    lds_barrier();
    int64_t before = 0, all = 0;
#pragma unroll
    for (int i = 0; i < kSerialWaves; ++i) {
        const int64_t x = tmp[i];
        if (i < wid) before = max64(before, x);
        all = max64(all, x);
    }
    *total = all;
    return max64(before, wave_shift_up1(incl, int64_t(0)));
}

// One decoder's peak inputs at step u: the stored prefix maximum, the floor
// of u's block, and the suffix maximum.
struct PeakIn {
    int64_t pf, fl, sa;
};

// Issued as three independent loads; the caller reads them once it needs them.
__device__ inline PeakIn peak_load(const CommitArgs& a, int32_t d, int32_t u) {
    const int64_t off = int64_t(d) * a.L + u;
    return PeakIn{a.PF[off], a.F[int64_t(d) * a.NB + u / kFloorBlock], a.SA[off]};
}

// Selection key of decoder d for the arrival (p, U): its peak and key.
__device__ inline int64_t commit_key(const PeakIn& in, int64_t p, int32_t C, int32_t Q, int32_t policy,
                                     int64_t* peak_out) {
    const int64_t peak = max64(p + max64(in.pf, in.fl), in.sa);
    const int64_t over = peak - C;
    *peak_out = peak;
    return (policy == MAPS_POLICY_MQ && over <= 0) ? int64_t(Q) - kFeasibleBias : over;
}

// Workgroup argmin of (key, d), lowest d on ties; every thread gets the
// result.  Wavefront minima by DPP, then one LDS round over the wavefronts.
__device__ inline void block_argmin(int64_t& key, int32_t& d, int64_t* skey, int32_t* sd) {
    const int64_t wk = wave_last(wave_incl_scan(key, INT64_MAX, [](int64_t x, int64_t y) { return x < y ? x : y; }));
    const int32_t wd =
        wave_last(wave_incl_scan(key == wk ? d : INT32_MAX, INT32_MAX,
                                 [](int32_t x, int32_t y) { return x < y ? x : y; }));
    const int lane = threadIdx.x % kWave, wid = threadIdx.x / kWave;
    if (lane == 0) { skey[wid] = wk; sd[wid] = wd; }
    lds_barrier();
    key = skey[0];
    d = sd[0];
    for (int i = 1; i < kSerialWaves; ++i)
        if (skey[i] < key || (skey[i] == key && sd[i] < d)) { key = skey[i]; d = sd[i]; }
}

// Values of the committed decoder at the next arrival's step, taken while
// its arrays are rewritten: the new PF there (next step <= U) and the new SA
// (next step < U).
struct Capture {
    int64_t pf, sa;
};

// Holds a loaded value in a register from this point on: the wait for its
// load is placed here, before the stores that follow (on gfx9 one counter
// covers loads and stores, so a later first use would also wait for those).
__device__ inline void pin(int64_t& x) { asm volatile("" : "+v"(x)); }

// Commit (p, Uc) to decoder bd: O += p + t on [0, Uc], PF and SA derived
// again there, and the new PF(Uc) recorded as a floor above Uc.  kStaged (a
// range of at most a.stage_cap entries): the new O values stay in LDS
// (`stage`) for the two scans; otherwise they are read back from HBM.  `un` is the next
// arrival's step (-1: none): the threads that rewrite PF(un) and SA(un) below
// Uc leave them in `cap`, and a thread with pre_d >= 0 loads decoder pre_d's
// peak inputs at un into *pre_out, issued with the range's loads.  Returns
// the new PF(Uc), the same in every thread.  Ends with a barrier after which
// every store of the commit is visible to the workgroup.
template <bool kStaged, typename SType = int64_t>
__device__ inline int64_t commit_range(const CommitArgs& a, SType* stage, int32_t bd, int64_t p, int32_t Uc,
                                       int32_t un, int32_t pre_d, PeakIn* pre_out, Capture* cap,
                                       int64_t* scan_tmp) {
    const int32_t L = a.L;
    const int lane = threadIdx.x % kWave, wid = threadIdx.x / kWave;
    int64_t* __restrict__ O = a.O + int64_t(bd) * L;
    int64_t* __restrict__ PF = a.PF + int64_t(bd) * L;
    int64_t* __restrict__ SA = a.SA + int64_t(bd) * L;
    int64_t* __restrict__ Fd = a.F + int64_t(bd) * a.NB;
    const int32_t n = Uc + 1;
    const int32_t chunk = (n + kSerialNT - 1) / kSerialNT;
    const int32_t b = threadIdx.x * chunk, e = b + chunk < n ? b + chunk : n;
    // above Uc: the rest of its block (up to kTailPer steps per thread) and
    // the block floors after it (up to kFloorPer per thread), read with the
    // range and raised to v last
    const int32_t kc = Uc / kFloorBlock;
    const int32_t tail_end = (kc + 1) * kFloorBlock < L ? (kc + 1) * kFloorBlock : L;
    int64_t tail_old[kTailPer];
#pragma unroll
    for (int k = 0; k < kTailPer; ++k) {
        const int32_t tt = Uc + 1 + int32_t(threadIdx.x) + k * kSerialNT;
        tail_old[k] = tt < tail_end ? PF[tt] : 0;
    }
    int64_t fb_old[kFloorPer];
#pragma unroll
    for (int k = 0; k < kFloorPer; ++k) {
        const int32_t blk = kc + 1 + int32_t(threadIdx.x) + k * kSerialNT;
        fb_old[k] = blk < a.NB ? Fd[blk] : 0;
    }
    int64_t sa_top = SA[Uc];   // max of O beyond Uc: unchanged by the commit
    const bool pre = un >= 0 && pre_d >= 0;
    PeakIn pl{0, 0, 0};
    if (pre) pl = peak_load(a, pre_d, un);
    int64_t mpre = 0, msuf = 0;
    int64_t o[kBatch];
    auto load_batch = [&](int32_t t0) {
#pragma unroll
        for (int j = 0; j < kBatch; ++j) o[j] = t0 + j < e ? O[t0 + j] : 0;
    };
    load_batch(b);
    // the loads issued before the range's are waited for now, ahead of its stores
    pin(sa_top);
    pin(pl.pf);
    pin(pl.fl);
    pin(pl.sa);
#pragma unroll
    for (int k = 0; k < kTailPer; ++k) pin(tail_old[k]);
#pragma unroll
    for (int k = 0; k < kFloorPer; ++k) pin(fb_old[k]);
    for (int32_t t0 = b; t0 < e; t0 += kBatch) {
        if (t0 != b) load_batch(t0);
#pragma unroll
        for (int j = 0; j < kBatch; ++j) {
            const int32_t t = t0 + j;
            if (t < e) {
                o[j] += p + t;
                O[t] = o[j];
                if constexpr (kStaged) stage[t] = SType(o[j]);
                mpre = max64(mpre, o[j] + t);
                msuf = max64(msuf, o[j]);
            }
        }
    }
    int64_t v;
    int64_t run = chain_excl_max(mpre, scan_tmp, &v);
    if (pre) *pre_out = pl;
    // suffix maxima over the chunks after this thread's (a scan in reversed thread order)
    int64_t incl = msuf;
    for (int k = 1; k < kWave; k <<= 1) {
        const int64_t x = __shfl_down(incl, k, kWave);
        if (lane + k < kWave) incl = max64(incl, x);
    }
    lds_barrier();   // every wave has read scan_tmp
    if (lane == 0) scan_tmp[wid] = incl;
    lds_barrier();
    int64_t after = sa_top;
#pragma unroll
    for (int w = 0; w < kSerialWaves; ++w)   // independent reads, one LDS round trip
        if (w > wid) after = max64(after, scan_tmp[w]);
    const int64_t below = __shfl_down(incl, 1, kWave);
    if (lane + 1 < kWave) after = max64(after, below);
    // the new O of the thread's entries [t0, t0 + kBatch), from LDS or HBM
    auto fetch = [&](int32_t t0, int64_t (&o)[kBatch]) {
        if constexpr (kStaged) {
#pragma unroll
            for (int j = 0; j < kBatch; ++j) o[j] = t0 + j < e ? int64_t(stage[t0 + j]) : 0;
        } else {
#pragma unroll
            for (int j = 0; j < kBatch; ++j) o[j] = t0 + j < e ? O[t0 + j] : 0;
        }
    };
    for (int32_t t0 = b; t0 < e; t0 += kBatch) {
        fetch(t0, o);
#pragma unroll
        for (int j = 0; j < kBatch; ++j) {
            const int32_t t = t0 + j;
            if (t < e) {
                run = max64(run, o[j] + t);
                PF[t] = run;
                if (t == un) cap->pf = run;
            }
        }
    }
    // SA from the top down, in batches [t1 - kBatch, t1)
    const int32_t last = b + ((e - b + kBatch - 1) / kBatch) * kBatch;   // past the thread's last batch
    for (int32_t t1 = last; t1 > b; t1 -= kBatch) {
        fetch(t1 - kBatch, o);
#pragma unroll
        for (int j = kBatch - 1; j >= 0; --j) {
            const int32_t t = t1 - kBatch + j;
            if (t < e) {
                if (t < Uc) {
                    SA[t] = after;
                    if (t == un) cap->sa = after;
                }
                after = max64(after, o[j]);
            }
        }
    }
    // the new PF(Uc) = v is a floor for every step above Uc
#pragma unroll
    for (int k = 0; k < kTailPer; ++k) {
        const int32_t tt = Uc + 1 + int32_t(threadIdx.x) + k * kSerialNT;
        if (tt < tail_end) PF[tt] = max64(tail_old[k], v);
    }
#pragma unroll
    for (int k = 0; k < kFloorPer; ++k) {
        const int32_t blk = kc + 1 + int32_t(threadIdx.x) + k * kSerialNT;
        if (blk < a.NB) Fd[blk] = max64(fb_old[k], v);
    }
    __syncthreads();
    return v;
}

// One workgroup for the whole chain.  kPre (D <= kSerialNT): thread d owns
// decoder d, and the next arrival's peak inputs are loaded while the current
// arrival is committed; only the committed decoder's inputs change, and its
// thread patches them from the values the commit captured.  Otherwise every
// thread evaluates its decoders d, d + kSerialNT, ... after each commit.
template <bool kPre>
__global__ __launch_bounds__(kSerialNT) void commit_serial(CommitArgs a) {
    extern __shared__ int32_t lds[];
    int32_t* Q = lds;                  // [D] running queue lengths
    int32_t* C = lds + a.S.D;          // [D] capacities
    int64_t* ostage = reinterpret_cast<int64_t*>(lds + 2 * a.S.D);   // [stage_cap] a commit's new O values
    __shared__ int32_t tile_p[2][kSerialNT], tile_U[2][kSerialNT];   // arrivals of the current and next tile
    __shared__ int64_t skey[kSerialWaves], scan_tmp[kSerialWaves];
    __shared__ int32_t sd[kSerialWaves];
    __shared__ int64_t speak;
    __shared__ Capture cap;
    const int32_t D = a.S.D, L = a.L, T = L - 1;
    const int tid = threadIdx.x;
    bool neg = false;
    for (int32_t d = tid; d < D; d += kSerialNT) {
        Q[d] = a.qlen[d];
        C[d] = a.cap[d];
        neg |= Q[d] < 0 || C[d] < 0;
    }
    if (neg) raise_error(a.dev_err, MAPS_ERR_NEG_LEN);
    auto stage = [&](int64_t tile) {   // arrivals of `tile` into its buffer
        const int64_t j = tile * kSerialNT + tid;
        tile_p[tile & 1][tid] = j < a.A ? a.ap[j] : 0;
        tile_U[tile & 1][tid] = j < a.A ? a.aU[j] : -1;
    };
    stage(0);
    __syncthreads();
    PeakIn cur{0, 0, 0};
    int64_t have = -1;   // the arrival whose inputs `cur` holds
    for (int64_t i = 0; i < a.A; ++i) {
        // the next tile is staged at the first arrival of a tile; the
        // barriers of that arrival precede every read of it
        if (i % kSerialNT == 0) stage(i / kSerialNT + 1);
        // uniform values read from LDS, made scalar so that every address derived from them is
        const int32_t p0 = __builtin_amdgcn_readfirstlane(tile_p[(i / kSerialNT) & 1][i % kSerialNT]);
        const int32_t U = __builtin_amdgcn_readfirstlane(tile_U[(i / kSerialNT) & 1][i % kSerialNT]);
        if (U < 0) {   // no bound: round robin, the request only joins the queue
            if (tid == 0) {
                const int32_t d = int32_t((a.rr_offset + i) % D);
                a.choice[i] = d;
                a.chosen_peak[i] = -1;
                a.chosen_over[i] = 0;
                a.flags[i] = 2;
                Q[d] += 1;
            }
            lds_barrier();
            continue;
        }
        if (tid == 0) {
            if (p0 < 0) raise_error(a.dev_err, MAPS_ERR_NEG_LEN);
            if (U > T) raise_error(a.dev_err, MAPS_ERR_BOUND_RANGE);
        }
        const int64_t p = p0 < 0 ? 0 : p0;
        const int32_t Uc = U < T ? U : T;
        // every decoder's peak with this arrival, and the thread's best key
        int64_t key = INT64_MAX, peak_best = 0;
        int32_t best = INT32_MAX;
        if constexpr (kPre) {
            if (tid < D) {
                if (have != i) cur = peak_load(a, tid, Uc);
                key = commit_key(cur, p, C[tid], Q[tid], a.policy, &peak_best);
                best = tid;
            }
        } else {
            for (int32_t d = tid; d < D; d += kSerialNT) {
                int64_t pk;
                const int64_t k = commit_key(peak_load(a, d, Uc), p, C[d], Q[d], a.policy, &pk);
                if (k < key) { key = k; best = d; peak_best = pk; }
            }
        }
        int64_t bkey = key;
        int32_t bd = best;
        block_argmin(bkey, bd, skey, sd);
        bd = __builtin_amdgcn_readfirstlane(bd);
        if (bd < 0 || bd >= D) bd = 0;   // unreachable with D >= 1; keeps every index in range
        if (best == bd && bd != INT32_MAX) speak = peak_best;   // the owner of the chosen decoder
        lds_barrier();
        const int64_t peak = speak;
        if (tid == 0) {
            const int64_t over = peak - C[bd];
            a.choice[i] = bd;
            a.chosen_peak[i] = peak;
            a.chosen_over[i] = over > 0 ? over : 0;
            a.flags[i] = over <= 0 ? 1 : 0;
            Q[bd] += 1;
        }
        // the next arrival's step, when it has a bound: its inputs go out with the commit's loads
        int32_t un = -1;
        if constexpr (kPre) {
            const int64_t j = i + 1;
            const int32_t Un =
                j < a.A ? __builtin_amdgcn_readfirstlane(tile_U[(j / kSerialNT) & 1][j % kSerialNT]) : -1;
            if (Un >= 0) un = Un < T ? Un : T;
        }
        const int32_t pre_d = kPre && tid < D ? tid : -1;
        // the new O values are at most peak + Uc (O(t) <= O(t) + t <= PF(Uc) <= peak - p, plus p + t): below
        // 2^31 they fit the stage as 32-bit values, twice as many of them
        const bool narrow = peak + Uc < int64_t(INT32_MAX);
        const int64_t v =
            Uc < a.stage_cap ? commit_range<true>(a, ostage, bd, p, Uc, un, pre_d, &cur, &cap, scan_tmp)
            : narrow && Uc < 2 * int64_t(a.stage_cap)
                ? commit_range<true, int32_t>(a, reinterpret_cast<int32_t*>(ostage), bd, p, Uc, un, pre_d, &cur,
                                              &cap, scan_tmp)
                : commit_range<false>(a, ostage, bd, p, Uc, un, pre_d, &cur, &cap, scan_tmp);
        if constexpr (kPre) {
            if (un >= 0) {
                if (tid < D) {
                    if (tid == bd) {   // rewritten on [0, Uc] (SA below Uc); above Uc, v is a floor
                        if (un <= Uc) cur.pf = cap.pf;
                        else cur.fl = max64(cur.fl, v);
                        if (un < Uc) cur.sa = cap.sa;
                    }
                }
                have = i + 1;
            }
        }
    }
    if (a.queue_out)
        for (int32_t d = tid; d < D; d += kSerialNT) a.queue_out[d] = Q[d];
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
    a.NB = c.NB;
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
    // dynamic LDS of the chain: queue lengths and capacities, then as many
    // staged range entries as the workgroup's LDS holds beside the kernel's
    // static LDS (less 256 bytes for the alignment of the dynamic part)
    auto serial = D <= kSerialNT ? commit_serial<true> : commit_serial<false>;
    const size_t qc = size_t(2) * D * sizeof(int32_t);   // a multiple of 8 bytes
    const size_t fixed = kernel_static_lds(serial) + qc + 256;
    if (fixed > kLdsPerWorkgroup) return MAPS_E_SIZE;   // unreachable with D <= MAPS_MAX_COMMIT_DECODERS
    a.stage_cap = int32_t((kLdsPerWorkgroup - fixed) / sizeof(int64_t));
    const size_t lds = qc + size_t(a.stage_cap) * sizeof(int64_t);
    hipLaunchKernelGGL(commit_init, dim3(unsigned(D)), dim3(kCommitNT), 0, stream, a);
    MAPS_CHECK_LAUNCH();
    allow_dynamic_lds(serial, lds);
    hipLaunchKernelGGL(serial, dim3(1), dim3(kSerialNT), lds, stream, a);
    MAPS_CHECK_LAUNCH();
    return MAPS_OK;
}
