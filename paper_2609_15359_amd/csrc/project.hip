// Projection of each decoder's KV occupancy (Sec. 3.3; App. A, Eq. (8)) on gfx950.
//
// One workgroup per decoder turns the residents' (prompt, generated, bound)
// triples into the snapshot described in maps_internal.hpp, without sorting:
//   1. every remaining length R = max(U - g, 0) sets its bit in a bitmap over
//      the step axis (LDS atomics);
//   2. an exclusive scan of the words' popcounts ranks the distinct R values:
//      the event index of R is the number of set bits below it;
//   3. residents add 1 and p + g to their event's counters (integer atomics,
//      so the sums are deterministic);
//   4. reverse scans give N_e and S_e, a forward max-scan the prefix maxima
//      PMX_e, a max-reduction the base peak;
//   5. when u_max is small enough, the dense profile F(u) for every u.
// Small decoders keep every array in LDS; decoders that do not fit run the
// same steps on their own slice of the snapshot in HBM.
#include "maps_internal.hpp"
#include "order_core.hpp"

namespace maps {
namespace {

constexpr int kNT = 1024;
constexpr size_t kLdsBudget = 150 * 1024;
constexpr int kResPer = 8;   // residents per thread held in registers (decoders of up to kNT * kResPer)
constexpr int kEvPer = 8;    // events per thread held in registers when the arrays are in LDS

// Arrays of one decoder: bitmap words, events before each word, and per event
// the count, the p+g sum, the time and the prefix maximum.
struct LdsArrays {
    uint32_t *bits, *wpre, *cnt, *wsum, *tau, *pmx;
    __device__ uint32_t& B(int64_t w) { return bits[w]; }
    __device__ uint32_t& P(int64_t w) { return wpre[w]; }
    __device__ uint32_t& C(int64_t e) { return cnt[e]; }
    __device__ uint32_t& S(int64_t e) { return wsum[e]; }
    __device__ uint32_t& T(int64_t e) { return tau[e]; }
    __device__ uint32_t& M(int64_t e) { return pmx[e]; }
    __device__ void events(uint32_t) {}
};

// The same arrays laid directly over the decoder's slice of the snapshot:
// rank word {bits, before}, PMX, tau -> T and the cold record {S, N} (the
// threshold and cold arrays are placed once the event count is known).
struct HbmArrays {
    uint32_t* rank;  // 2 words per rank entry
    uint32_t* pmx;   // 1 word per event
    uint32_t* thr;   // 1 word per event
    uint32_t* cold;  // 2 words per cold record
    __device__ uint32_t& B(int64_t w) { return rank[2 * w]; }
    __device__ uint32_t& P(int64_t w) { return rank[2 * w + 1]; }
    __device__ uint32_t& M(int64_t e) { return pmx[e]; }
    __device__ uint32_t& T(int64_t e) { return thr[e]; }
    __device__ uint32_t& S(int64_t e) { return cold[2 * e]; }
    __device__ uint32_t& C(int64_t e) { return cold[2 * e + 1]; }
    __device__ void events(uint32_t E) {
        thr = pmx + 4 * event_units(E);
        cold = thr + 4 * event_units(E);
    }
};

__device__ inline int64_t remaining(int32_t U, int32_t g) {
    int64_t R = int64_t(U) - g;
    return R > 0 ? R : 0;
}

// Phase boundary: every thread's writes of the previous phase are visible to
// the whole workgroup.  For arrays in HBM each thread first waits until its
// own stores and atomics have reached L2, and after the barrier drops its
// vector-L1 lines, since values produced by L2 atomics may be cached stale
// (the slice is this workgroup's alone: no L2 write-back is needed).
template <bool kInLds>
__device__ inline void phase() {
    if constexpr (!kInLds) __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if constexpr (!kInLds) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
}

struct Scratch {
    int64_t red64[kNT / kWave];
    uint32_t red32[kNT / kWave];
    int4 red4[kNT / kWave];
};

// Four workgroup-wide maxima at once (one LDS round instead of four), and a
// sum when `sum` is given.  Without kGuard the caller guarantees that no
// thread still reads `tmp` or `tmp_sum` from an earlier use.
template <bool kGuard = true>
__device__ inline int4 block_reduce_max4(int4 v, int4* tmp, int64_t* sum = nullptr, int64_t* tmp_sum = nullptr) {
    v.x = wave_reduce_max(v.x);
    v.y = wave_reduce_max(v.y);
    v.z = wave_reduce_max(v.z);
    v.w = wave_reduce_max(v.w);
    const int lane = threadIdx.x % kWave, wid = threadIdx.x / kWave;
    int64_t s = 0;
    if (sum) s = wave_reduce_add(*sum);
    if constexpr (kGuard) __syncthreads();
    if (lane == 0) {
        tmp[wid] = v;
        if (sum) tmp_sum[wid] = s;
    }
    __syncthreads();
    if (sum) {
        s = 0;
#pragma unroll
        for (int i = 0; i < kNT / kWave; ++i) s += tmp_sum[i];
        *sum = s;
    }
    int4 r = tmp[0];
#pragma unroll
    for (int i = 1; i < kNT / kWave; ++i) {
        const int4 t = tmp[i];
        r.x = r.x > t.x ? r.x : t.x;
        r.y = r.y > t.y ? r.y : t.y;
        r.z = r.z > t.z ? r.z : t.z;
        r.w = r.w > t.w ? r.w : t.w;
    }
    return r;
}

// kRP residents and kEP events per thread in registers: (4, 4) for decoders
// of at most 4 * kNT residents (fewer instructions in every unrolled loop),
// (8, 8) otherwise.
template <bool kInLds, int kRP, int kEP, typename Arr>
__device__ void project_one(Arr a, int32_t d, int64_t lo, int64_t hi, const int32_t* __restrict__ p,
                            const int32_t* __restrict__ g, const int32_t* __restrict__ U, int32_t u_max, int32_t W,
                            int32_t P, SnapView V, int64_t slice_off, int32_t* __restrict__ base_peak, uint32_t* dev_err,
                            Scratch& sc, DecHeader* hdr_out) {
    const int tid = threadIdx.x;
    for (int64_t w = tid; w < W; w += kNT) a.B(w) = 0u;
    if constexpr (kInLds) {   // the event counters too: E <= residents <= the LDS capacity
        for (int64_t e = tid; e < hi - lo; e += kNT) { a.C(e) = 0u; a.S(e) = 0u; }
    }
    phase<kInLds>();

    // 1. event bitmap and total demand sum_r (p + g + R).  A decoder of at
    // most kNT * kRP residents is read once, every load in flight
    // together, and keeps R and p + g in registers for step 3.
    int64_t tot = 0;
    bool neg = false, range = false;
    const int64_t n = hi - lo;
    const bool in_regs = n <= int64_t(kNT) * kRP;
    uint32_t Rk[kRP], PGk[kRP];
    auto resident = [&](int32_t pr, int32_t gr, int32_t ur, uint32_t& Rout, uint32_t& PGout) {
        neg |= (pr < 0) | (gr < 0) | (ur < 0);
        pr = pr < 0 ? 0 : pr;
        gr = gr < 0 ? 0 : gr;
        int64_t R = remaining(ur < 0 ? 0 : ur, gr);
        if (R > u_max) { range = true; R = u_max; }
        atomicOr(&a.B(R >> 5), 1u << (R & 31));
        tot += int64_t(pr) + gr + R;
        Rout = uint32_t(R);
        PGout = uint32_t(pr) + uint32_t(gr);
    };
    if (in_regs) {
        int32_t pr[kRP], gr[kRP], ur[kRP];
#pragma unroll
        for (int j = 0; j < kRP; ++j) {
            const int64_t i = int64_t(j) * kNT + tid;
            pr[j] = i < n ? p[lo + i] : 0;
            gr[j] = i < n ? g[lo + i] : 0;
            ur[j] = i < n ? U[lo + i] : 0;
        }
#pragma unroll
        for (int j = 0; j < kRP; ++j) {
            Rk[j] = 0u;
            PGk[j] = 0u;
            if (int64_t(j) * kNT + tid < n) resident(pr[j], gr[j], ur[j], Rk[j], PGk[j]);
        }
    } else {
        for (int64_t r = lo + tid; r < hi; r += kNT) {
            uint32_t R, PG;
            resident(p[r], g[r], U[r], R, PG);
        }
    }
    if (neg) raise_error(dev_err, MAPS_ERR_NEG_LEN);
    if (range) raise_error(dev_err, MAPS_ERR_BOUND_RANGE);
    if constexpr (!kInLds) {   // the LDS path sums the demand with its last reduction
        tot = block_reduce_add<kNT>(tot, sc.red64);
        if (tid == 0 && tot + u_max > int64_t(INT32_MAX)) raise_error(dev_err, MAPS_ERR_INT32_RANGE);
    }
    phase<kInLds>();

    // 2. events before each bitmap word
    const uint32_t E = block_scan<kNT, false, false, true, uint32_t>(
        W, 0u, [&](int64_t w) { return uint32_t(__popc(a.B(w))); },
        [&](int64_t w, uint32_t v) { a.P(w) = v; }, sc.red32);   // ends with a barrier
    a.events(E);
    if constexpr (!kInLds) phase<kInLds>();

    // 3. per-event counters (in LDS already zero, and independent of the
    //    event times: no barrier between the two loops)
    if constexpr (!kInLds) {
        for (int64_t e = tid; e < E; e += kNT) { a.C(e) = 0u; a.S(e) = 0u; }
    }
    for (int64_t w = tid; w < W; w += kNT) {       // event times, in rank order
        uint32_t bits = a.B(w), e = a.P(w);
        while (bits) {
            a.T(e++) = uint32_t(w * 32 + (__ffs(bits) - 1));
            bits &= bits - 1u;
        }
    }
    if constexpr (!kInLds) phase<kInLds>();
    auto count = [&](uint32_t R, uint32_t PG) {
        const uint32_t word = a.B(R >> 5);
        const uint32_t e = a.P(R >> 5) + __popc(word & ((1u << (R & 31)) - 1u));
        atomicAdd(&a.C(e), 1u);
        atomicAdd(&a.S(e), PG);
    };
    if (in_regs) {
#pragma unroll
        for (int j = 0; j < kRP; ++j)
            if (int64_t(j) * kNT + tid < n) count(Rk[j], PGk[j]);
    } else {
        for (int64_t r = lo + tid; r < hi; r += kNT) {
            int32_t pr = p[r], gr = g[r], ur = U[r];
            pr = pr < 0 ? 0 : pr;
            gr = gr < 0 ? 0 : gr;
            int64_t R = remaining(ur < 0 ? 0 : ur, gr);
            if (R > u_max) R = u_max;
            count(uint32_t(R), uint32_t(pr) + uint32_t(gr));
        }
    }
    phase<kInLds>();

    // 4. N_e and S_e: suffix sums over the events (of N << 32 | S: S stays
    //    below 2^32, a larger total demand is reported as out of range); then
    //    PMX_e = max(0, max_{i<e} S_i + tau_i (N_i + 1)) by a forward max-scan;
    //    then the base peak max(0, max_e S_e + tau_e N_e), the thresholds T_e,
    //    the hot window (bounds above event 0's cold range and below the first
    //    cold range of a later event, [max(T_e, tau_{e-1} + 1), tau_e] for
    //    e < E: the last event needs no cold record) and the flat region
    //    (bounds past the first event e* with PMX_e = PMX_E, i.e.
    //    U >= tau_{e*-1} + 1).
    int32_t pmx_end, bmax = 0, lo_w = 0, start_min = INT32_MAX, estar = int32_t(E);
    // the snapshot slice: rank words, then PMX_e, T_e and the cold records {S_e, N_e + 1}
    uint2* rank = reinterpret_cast<uint2*>(V.slices + slice_off);
    int32_t* pmx = reinterpret_cast<int32_t*>(V.slices + slice_off + W / 2);
    int32_t* thr = pmx + 4 * event_units(E);
    int2* cold = reinterpret_cast<int2*>(thr + 4 * event_units(E));
    // register chunks of the LDS path: after the pass below, per event the
    // suffix count N_e (cN), the suffix sum S_e (cS), the threshold T_e (cT)
    // and PMX_e (cM)
    uint32_t cN[kEP], cS[kEP], cT[kEP];
    int32_t cM[kEP];
    bool ok[kEP];
    const int chunk = int((int64_t(E) + kNT - 1) / kNT);
    const int e0 = kInLds ? tid * chunk : 0;
    if constexpr (kInLds) {
        // E <= residents <= kNT * kEP: each thread keeps its contiguous
        // chunk of events in registers through both scans and the thresholds
#pragma unroll
        for (int j = 0; j < kEP; ++j) {
            const int e = e0 + j;
            ok[j] = j < chunk && e < int(E);
            cN[j] = ok[j] ? a.C(e) : 0u;
            cS[j] = ok[j] ? a.S(e) : 0u;
            cT[j] = ok[j] ? a.T(e) : 0u;
        }
        uint64_t loc = 0;
#pragma unroll
        for (int j = 0; j < kEP; ++j) loc += (uint64_t(cN[j]) << 32) | cS[j];
        uint64_t all;
        const uint64_t before =
            block_excl_scan<kNT, false, uint64_t, false>(loc, uint64_t(0), reinterpret_cast<uint64_t*>(sc.red64), &all);
        uint64_t run = all - before - loc;   // the events after this chunk
        int32_t v[kEP];
        int32_t lmax = 0;
#pragma unroll
        for (int j = kEP - 1; j >= 0; --j) {
            run += (uint64_t(cN[j]) << 32) | cS[j];
            cN[j] = uint32_t(run >> 32);
            cS[j] = uint32_t(run);
            v[j] = int32_t(cS[j] + cT[j] * (cN[j] + 1u));
            if (ok[j]) lmax = lmax > v[j] ? lmax : v[j];
        }
        int32_t mall;
        // red32 was last read before the barriers of the scan above
        int32_t m = block_excl_scan<kNT, true, int32_t, false>(lmax, 0, reinterpret_cast<int32_t*>(sc.red32), &mall);
        pmx_end = mall;
        uint32_t prev_tau = e0 >= 1 && e0 - 1 < int(E) ? a.T(e0 - 1) : 0u;
#pragma unroll
        for (int j = 0; j < kEP; ++j) {
            cM[j] = m;
            if (!ok[j]) continue;
            const int e = e0 + j;
            const int32_t o = int32_t(cS[j] + cT[j] * cN[j]);
            bmax = bmax > o ? bmax : o;
            if (m == pmx_end && e < estar) estar = e;
            const int32_t T = event_threshold(m, int32_t(cS[j]), cN[j] + 1u);
            if (P > 0) {   // the dense profile reads the scanned arrays back
                a.C(e) = cN[j];
                a.S(e) = cS[j];
                a.M(e) = uint32_t(m);
            }
            const int64_t lo_e = e == 0 ? 0 : int64_t(prev_tau) + 1;
            const int64_t hi_e = int64_t(cT[j]);
            const int64_t start = T > lo_e ? T : lo_e;
            if (start <= hi_e) {   // a bound landing on e reaches T_e
                if (e == 0) lo_w = int32_t(hi_e + 1);
                else if (start < start_min) start_min = int32_t(start);
            }
            prev_tau = cT[j];
            cT[j] = uint32_t(T);
            m = m > v[j] ? m : v[j];
        }
    } else {
        block_scan<kNT, false, true, false, uint64_t>(
            E, uint64_t(0), [&](int64_t e) { return (uint64_t(a.C(e)) << 32) | a.S(e); },
            [&](int64_t e, uint64_t v) {
                a.C(e) = uint32_t(v >> 32);
                a.S(e) = uint32_t(v);
            },
            reinterpret_cast<uint64_t*>(sc.red64));
        phase<kInLds>();
        pmx_end = block_scan<kNT, true, false, true, int32_t>(
            E, 0,
            [&](int64_t e) { return int32_t(a.S(e) + a.T(e) * (a.C(e) + 1u)); },
            [&](int64_t e, int32_t v) { a.M(e) = uint32_t(v); }, reinterpret_cast<int32_t*>(sc.red32));
        phase<kInLds>();
        for (int64_t e = tid; e < E; e += kNT) {
            const int32_t o = int32_t(a.S(e) + a.T(e) * a.C(e));
            bmax = bmax > o ? bmax : o;
            const int32_t m = int32_t(a.M(e));
            if (m == pmx_end && int32_t(e) < estar) estar = int32_t(e);
            const int64_t T = event_threshold(m, int32_t(a.S(e)), a.C(e) + 1u);
            const int64_t lo_e = e == 0 ? 0 : int64_t(a.T(e - 1)) + 1;
            const int64_t hi_e = int64_t(a.T(e));
            const int64_t start = T > lo_e ? T : lo_e;
            if (start > hi_e) continue;   // no bound landing on e reaches T_e
            if (e == 0) lo_w = int32_t(hi_e + 1);
            else if (start < start_min) start_min = int32_t(start);
        }
    }
    int4 r;
    if constexpr (kInLds) {   // red4 unused so far, red64 last read before the barriers of the max-scan
        r = block_reduce_max4<false>(make_int4(bmax, lo_w, -start_min, -estar), sc.red4, &tot, sc.red64);
        if (tid == 0 && tot + u_max > int64_t(INT32_MAX)) raise_error(dev_err, MAPS_ERR_INT32_RANGE);
    } else {
        r = block_reduce_max4(make_int4(bmax, lo_w, -start_min, -estar), sc.red4);
    }
    const int32_t base = r.x, hot_lo = r.y, hot_hi = -r.z - 1, e_star = -r.w;
    const int32_t flat_lo = e_star == 0 ? 0 : int32_t(a.T(e_star - 1)) + 1;

    // 5. dense profile F(u) = max(PMX_e, S_e + u (N_e + 1), u), e = #{events < u}
    if (P > 0) {
        int32_t* prof = V.prof + int64_t(d) * P;
        for (int64_t u = tid; u < P; u += kNT) {
            const uint32_t word = a.B(u >> 5);
            const uint32_t e = a.P(u >> 5) + __popc(word & ((1u << (u & 31)) - 1u));
            int32_t pm = pmx_end, lin = int32_t(u);
            if (e < E) {
                pm = int32_t(a.M(e));
                lin = int32_t(a.S(e) + uint32_t(u) * (a.C(e) + 1u));
            }
            const int32_t f = pm > lin ? pm : lin;
            prof[u] = f > int32_t(u) ? f : int32_t(u);
        }
        phase<kInLds>();   // the HBM arrays are updated in place below
    }

    // 6. the rest of the snapshot slice (arrays in LDS: the rank words; in
    //    HBM: T_e and N_e + 1 in place)
    if constexpr (kInLds) {
        // the event arrays from the registers, after the last barrier (a
        // barrier waits for every store in flight)
#pragma unroll
        for (int j = 0; j < kEP; ++j) {
            if (!ok[j]) continue;
            const int e = e0 + j;
            pmx[e] = cM[j];
            thr[e] = int32_t(cT[j]);
            cold[e] = make_int2(int32_t(cS[j]), int32_t(cN[j] + 1u));
        }
        for (int64_t w = tid; w < W; w += kNT) rank[w] = make_uint2(a.B(w), a.P(w));
    } else {
        for (int64_t e = tid; e < E; e += kNT) {   // in place: each thread owns its events
            const uint32_t n1 = a.C(e) + 1u;
            a.T(e) = uint32_t(event_threshold(int32_t(a.M(e)), int32_t(a.S(e)), n1));
            a.C(e) = n1;
        }
    }
    if (tid == 0) {
        pmx[E] = pmx_end;
        thr[E] = event_threshold(pmx_end, 0, 1u);
        cold[E] = make_int2(0, 1);
        DecHeader h;
        h.slice_off = slice_off;
        h.tot = tot;
        h.E = int32_t(E);
        h.base_peak = base;
        h.hot_lo = hot_lo;
        h.hot_hi = hot_hi;
        h.flat_lo = flat_lo;
        h.pmx_end = pmx_end;
        for (int i = 0; i < 6; ++i) h.pad[i] = 0;
        V.dec[d] = h;
        if (hdr_out != nullptr) *hdr_out = h;
        base_peak[d] = base;
    }
}

// Decoder d's projection (the slice, its header and base peak) by one
// workgroup of kNT threads; `lds` is the launch's dynamic LDS.
// [lo, hi): the decoder's residents (seg_off[d], seg_off[d + 1], loaded by the
// caller); hdr_out (nullable, LDS): receives the decoder header written.
__device__ inline void project_decoder(int32_t d, int32_t D, int64_t lo, int64_t hi, int64_t n_total,
                                       const int32_t* __restrict__ p, const int32_t* __restrict__ g,
                                       const int32_t* __restrict__ U, int32_t u_max, const SnapLayout& L,
                                       void* snap, int32_t* __restrict__ base_peak, int64_t lds_cap,
                                       uint32_t* dev_err, uint32_t* lds, DecHeader* hdr_out = nullptr) {
    __shared__ Scratch sc;
    const int32_t W = L.W;
    SnapView V = snap_view(snap, L);
    if (!(0 <= lo && lo <= hi && hi <= n_total)) {
        if (threadIdx.x == 0) raise_error(dev_err, MAPS_ERR_SEG_OFFSETS);
        lo = lo < 0 ? 0 : (lo > n_total ? n_total : lo);
        hi = lo;
    }
    if (hi - lo >= MAPS_MAX_RESIDENTS) {
        if (threadIdx.x == 0) raise_error(dev_err, MAPS_ERR_TOO_MANY);
        hi = lo;
    }
    // decoder d's slice: W/2 units of rank words, then the event arrays (at most hi - lo + kSliceSpare units)
    const int64_t slice_off = lo + int64_t(d) * (kSliceSpare + W / 2);
    if (d == 0 && threadIdx.x == 0) {   // the snapshot header: every field is known before the decoders
        SnapHeader h;
        h.D = D;
        h.u_max = u_max;
        h.W = W;
        h.n_total = n_total;
        h.P = L.P;
        for (int i = 0; i < 9; ++i) h.pad[i] = 0;
        h.magic = kSnapMagic;
        *V.hdr = h;
    }
    if (lds_cap > 0 && hi - lo <= lds_cap) {
        LdsArrays a;
        a.bits = lds;
        a.wpre = lds + W;
        a.cnt = lds + 2 * W;
        a.wsum = a.cnt + lds_cap;
        a.tau = a.wsum + lds_cap;
        a.pmx = a.tau + lds_cap;
        if (hi - lo <= int64_t(kNT) * 4)
            project_one<true, 4, 4>(a, d, lo, hi, p, g, U, u_max, W, L.P, V, slice_off, base_peak, dev_err, sc,
                                    hdr_out);
        else
            project_one<true, kResPer, kEvPer>(a, d, lo, hi, p, g, U, u_max, W, L.P, V, slice_off, base_peak,
                                               dev_err, sc, hdr_out);
    } else {
        HbmArrays a;
        a.rank = reinterpret_cast<uint32_t*>(V.slices + slice_off);
        a.pmx = reinterpret_cast<uint32_t*>(V.slices + slice_off + W / 2);
        a.thr = nullptr;
        a.cold = nullptr;
        project_one<false, kResPer, kEvPer>(a, d, lo, hi, p, g, U, u_max, W, L.P, V, slice_off, base_peak, dev_err,
                                            sc, hdr_out);
    }
}

__global__ __launch_bounds__(kNT) void project_decoders(int32_t D, const int64_t* __restrict__ seg_off,
                                                        int64_t n_total, const int32_t* __restrict__ p,
                                                        const int32_t* __restrict__ g,
                                                        const int32_t* __restrict__ U, int32_t u_max,
                                                        SnapLayout L, void* snap, int32_t* __restrict__ base_peak,
                                                        int64_t lds_cap, uint32_t* dev_err) {
    extern __shared__ uint32_t lds[];
    const int32_t d = int32_t(blockIdx.x);
    project_decoder(d, D, seg_off[d], seg_off[d + 1], n_total, p, g, U, u_max, L, snap, base_peak, lds_cap,
                    dev_err, lds);
}

// Projection and local order in one launch: workgroup d projects decoder d,
// then (once its slice and header are stored) orders d's queue against that
// slice, in the same dynamic LDS.  The order's latency-bound work then costs
// no launch and no pass of its own.
static_assert(order::kOrderNT == kNT, "one workgroup size for both steps");
__global__ __launch_bounds__(kNT) void project_order_decoders(int32_t D, const int64_t* __restrict__ seg_off,
                                                              int64_t n_total, const int32_t* __restrict__ p,
                                                              const int32_t* __restrict__ g,
                                                              const int32_t* __restrict__ U, int32_t u_max,
                                                              SnapLayout L, void* snap,
                                                              int32_t* __restrict__ base_peak, int64_t lds_cap,
                                                              uint32_t* dev_err, order::LocalArgs o) {
    extern __shared__ uint32_t lds[];
    __shared__ DecHeader hdr;
    const int32_t d = int32_t(blockIdx.x);
    // the residents' offsets and the queue's inputs are loaded together
    // first, so the queue's loads are in flight during the projection
    const int64_t lo = seg_off[d], hi = seg_off[d + 1];
    const order::QueueFetch qf = order::fetch_queue(o, d);
    project_decoder(d, D, lo, hi, n_total, p, g, U, u_max, L, snap, base_peak, lds_cap, dev_err, lds, &hdr);
    __syncthreads();   // the slice and header stores of this workgroup are done; hdr holds the header
    order::order_queue(o, d, n_total, &hdr, &qf);
}

}  // namespace
}  // namespace maps

using namespace maps;

extern "C" size_t maps_snapshot_bytes(int32_t D, int64_t n_total, int32_t u_max) {
    if (D < 1 || n_total < 0 || u_max < 0 || u_max > MAPS_MAX_U_MAX) return 0;
    return snap_layout(D, n_total, u_max).bytes;
}

extern "C" size_t maps_project_workspace_size(int32_t, int64_t, int32_t) { return 0; }

extern "C" maps_status maps_project(int32_t D, const int64_t* seg_off, int64_t n_total,
                                    const int32_t* prompt, const int32_t* generated, const int32_t* upper,
                                    int32_t u_max, void* snapshot, size_t snapshot_bytes, int32_t* base_peak,
                                    uint32_t* dev_err, void* workspace, size_t workspace_bytes,
                                    hipStream_t stream) {
    (void)workspace;
    (void)workspace_bytes;
    if (D < 1 || n_total < 0 || u_max < 0 || u_max > MAPS_MAX_U_MAX) return MAPS_E_SIZE;
    if (!seg_off || !snapshot || !base_peak || !dev_err ||
        (n_total > 0 && (!prompt || !generated || !upper)))
        return MAPS_E_NULL;
    const SnapLayout L = snap_layout(D, n_total, u_max);
    if (snapshot_bytes < L.bytes) return MAPS_E_BUFFER;
    const size_t fixed = size_t(2) * L.W * 4;
    int64_t cap = fixed < kLdsBudget ? int64_t((kLdsBudget - fixed) / 16) : 0;
    if (cap > int64_t(kNT) * kEvPer) cap = int64_t(kNT) * kEvPer;   // the register chunks of the LDS path
    const size_t lds = cap > 0 ? fixed + size_t(cap) * 16 : 0;
    allow_dynamic_lds(project_decoders, lds);
    hipLaunchKernelGGL(project_decoders, dim3(D), dim3(kNT), lds, stream, D, seg_off, n_total, prompt, generated,
                       upper, u_max, L, snapshot, base_peak, cap, dev_err);
    MAPS_CHECK_LAUNCH();
    return MAPS_OK;
}

extern "C" maps_status maps_project_order(int32_t D, const int64_t* seg_off, int64_t n_total,
                                          const int32_t* prompt, const int32_t* generated, const int32_t* upper,
                                          int32_t u_max, void* snapshot, size_t snapshot_bytes, int32_t* base_peak,
                                          const int32_t* capacity, const int64_t* q_off, int64_t q_total,
                                          const int32_t* q_prompt, const int32_t* q_upper, const int32_t* q_wait_ms,
                                          int32_t max_wait_ms, int32_t* order, int32_t* admitted,
                                          uint32_t* dev_err, hipStream_t stream) {
    if (D < 1 || n_total < 0 || q_total < 0 || u_max < 0 || u_max > MAPS_MAX_U_MAX) return MAPS_E_SIZE;
    if (!seg_off || !snapshot || !base_peak || !dev_err || !capacity || !q_off || !admitted ||
        (n_total > 0 && (!prompt || !generated || !upper)) || (q_total > 0 && (!q_prompt || !q_upper || !order)))
        return MAPS_E_NULL;
    const SnapLayout L = snap_layout(D, n_total, u_max);
    if (snapshot_bytes < L.bytes) return MAPS_E_BUFFER;
    // the local order's LDS is static, beside the projection's: a smaller
    // budget for the projection's arrays (larger decoders run from HBM)
    constexpr size_t kFusedBudget = kLdsBudget - sizeof(order::LocalLds);
    const size_t fixed = size_t(2) * L.W * 4;
    int64_t cap = fixed < kFusedBudget ? int64_t((kFusedBudget - fixed) / 16) : 0;
    if (cap > int64_t(kNT) * kEvPer) cap = int64_t(kNT) * kEvPer;
    const size_t lds = cap > 0 ? fixed + size_t(cap) * 16 : 0;
    order::LocalArgs o;
    o.L = L;
    o.snap = snapshot;
    o.cap = capacity;
    o.q_off = q_off;
    o.total = q_total;
    o.qp = q_prompt;
    o.qU = q_upper;
    o.qwait = q_wait_ms;
    o.max_wait = max_wait_ms;
    o.order = order;
    o.admitted = admitted;
    o.dev_err = dev_err;
    allow_dynamic_lds(project_order_decoders, lds);
    hipLaunchKernelGGL(project_order_decoders, dim3(D), dim3(kNT), lds, stream, D, seg_off, n_total, prompt,
                       generated, upper, u_max, L, snapshot, base_peak, cap, dev_err, o);
    MAPS_CHECK_LAUNCH();
    return MAPS_OK;
}
