#pragma once
// Local SJF order and admission (Sec. 3.3, Eq. (7); App. A, Eq. (10)) on gfx950:
// the device code, shared by the local-order launch and the launch that ends
// placement and orders every local queue.
//
// One workgroup per decoder:
//   1. bitonic sort in LDS of the packed keys (promoted?0:1, promoted? index :
//      bound, index) -- unique keys, so the order is the stable one;
//   2. a second bitonic sort of (bound, index) gives the queue by bound, with
//      the start of each run of equal bounds;
//   (a queue of at most 64 requests is ordered by counting instead, each
//   wavefront counting against 4 of its requests);
//   3. admitted = the largest k whose prefix keeps the projected peak within
//      the capacity, by binary search over k (the peak never decreases when a
//      request is added).  For a prefix, residents plus admitted requests form
//      a curve that increases between breakpoints -- the residents' event
//      times and the requests' bounds -- so the peak is its maximum over those
//      points.  At a point t the prefix contributes sum (p_i + t) over members
//      with bound >= t: masked suffix sums over the bound-sorted queue give it
//      in O(1) after one scan per k.  Residents' occupancy comes from the
//      snapshot (record S + t N at the rank of t).
#include "maps_internal.hpp"

namespace maps {
namespace order {

constexpr int kOrderNT = 1024;
constexpr int kMaxQ = MAPS_MAX_LOCAL_QUEUE;

struct LocalArgs {
    SnapLayout L;
    const void* snap;
    const int32_t* cap;
    const int64_t* q_off;
    int64_t total;
    const int32_t* qp;
    const int32_t* qU;
    const int32_t* qwait;
    int32_t max_wait;
    int32_t* order;
    int32_t* admitted;
    uint32_t* dev_err;
};

struct LocalLds {
    // the sort keys (steps 1-2) and the prompt suffix sums (step 3) are never
    // live together: sharing their space leaves room for two workgroups per CU
    union {
        uint64_t keys[kMaxQ];
        int64_t psuf[kMaxQ + 1];  // prompts summed over the members csuf counts
    };
    int32_t pos[kMaxQ];       // position of queue entry i in the new order
    int32_t ue[kMaxQ];        // bound of entry i (missing bound -> u_max)
    int32_t pp[kMaxQ];        // prompt of entry i
    int32_t uidx[kMaxQ];      // entries sorted by (bound, index)
    int32_t grp[kMaxQ];       // first position of the run of equal bounds
    int32_t csuf[kMaxQ + 1];  // members of the prefix with bound >= that position's bound
    int64_t red64[kOrderNT / kWave];
    int32_t red32[kOrderNT / kWave];
};

__device__ inline void bitonic_sort(uint64_t* keys, int n2) {
    for (int k = 2; k <= n2; k <<= 1) {
        for (int j = k >> 1; j > 0; j >>= 1) {
            for (int i = threadIdx.x; i < n2; i += kOrderNT) {
                const int ixj = i ^ j;
                if (ixj > i) {
                    const uint64_t a = keys[i], b = keys[ixj];
                    const bool up = (i & k) == 0;
                    if ((a > b) == up) { keys[i] = b; keys[ixj] = a; }
                }
            }
            __syncthreads();
        }
    }
}

// Largest projected peak of the residents plus the first k requests of the new order.
__device__ inline int64_t prefix_peak(LocalLds& s, int n, int k, const uint2* rank, const int2* cold, int32_t E,
                               int32_t W) {
    block_scan<kOrderNT, false, true, false, int32_t>(
        n, 0, [&](int64_t i) { return int32_t(s.pos[s.uidx[i]] < k); },
        [&](int64_t i, int32_t v) { s.csuf[i] = v; }, s.red32);
    block_scan<kOrderNT, false, true, false, int64_t>(
        n, int64_t(0), [&](int64_t i) { const int j = s.uidx[i]; return s.pos[j] < k ? int64_t(s.pp[j]) : int64_t(0); },
        [&](int64_t i, int64_t v) { s.psuf[i] = v; }, s.red64);
    if (threadIdx.x == 0) { s.csuf[n] = 0; s.psuf[n] = 0; }
    __syncthreads();
    int64_t best = 0;
    // resident event times: the set bits of the rank words, event e the
    // (before + j)-th of them
    for (int w = threadIdx.x; w < W; w += kOrderNT) {
        const uint2 rw = rank[w];
        uint32_t bits = rw.x, e = rw.y;
        for (; bits != 0u && e < uint32_t(E); bits &= bits - 1u, ++e) {
            const int64_t tau = int64_t(w) * 32 + (__ffs(bits) - 1);
            const int2 r = cold[e];
            int lo = 0, hi = n;   // first bound-sorted position with bound >= tau
            while (lo < hi) {
                const int mid = (lo + hi) >> 1;
                if (s.ue[s.uidx[mid]] < tau) lo = mid + 1; else hi = mid;
            }
            const int64_t v = int64_t(r.x) + tau * (r.y - 1) + s.psuf[lo] + tau * s.csuf[lo];
            best = best > v ? best : v;
        }
    }
    // bounds of the admitted requests
    const int32_t ucl_max = 32 * W - 1;
    for (int i = threadIdx.x; i < n; i += kOrderNT) {
        const int j = s.uidx[i];
        if (s.pos[j] >= k) continue;
        const int64_t t = s.ue[j];
        const int32_t tc = t < ucl_max ? int32_t(t) : ucl_max;
        const uint2 w = rank[tc >> 5];
        uint32_t e = w.y + __popc(w.x & ((1u << (tc & 31)) - 1u));
        e = e < uint32_t(E) ? e : uint32_t(E);
        const int2 r = cold[e];
        const int64_t occ = e < uint32_t(E) ? int64_t(r.x) + t * (r.y - 1) : 0;
        const int g0 = s.grp[i];
        const int64_t v = occ + s.psuf[g0] + t * s.csuf[g0];
        best = best > v ? best : v;
    }
    return block_reduce_max<kOrderNT>(best, s.red64);
}

// Decoder d's queue bounds and capacity, and, when the queue holds at most
// one wavefront of requests, request i's prompt, bound and wait in lane i of
// every wavefront (0 elsewhere).  Called early by a launch that has other work first, so
// that these loads are in flight during it.
struct QueueFetch {
    int64_t qlo, qhi;
    int32_t C, pr, u, wait;
};

__device__ inline QueueFetch fetch_queue(const LocalArgs& g, int32_t d) {
    QueueFetch f;
    f.qlo = g.q_off[d];
    f.qhi = g.q_off[d + 1];
    f.C = g.cap[d];
    f.pr = 0;
    f.u = 0;
    f.wait = 0;
    const int64_t i = f.qlo + int64_t(threadIdx.x % kWave);   // every wavefront holds the short queue
    if (0 <= f.qlo && f.qlo <= f.qhi && f.qhi <= g.total && f.qhi - f.qlo <= kWave && i < f.qhi) {
        f.pr = g.qp[i];
        f.u = g.qU[i];
        f.wait = g.qwait != nullptr ? g.qwait[i] : 0;
    }
    return f;
}

// The whole local order of decoder d by one workgroup of kOrderNT threads.
// built != nullptr: the snapshot's decoder d was written by this workgroup
// (the projection's launch), which passes the header it wrote (the
// snapshot's own header, written by another workgroup, cannot be read back
// reliably) and the resident count.  pre (nullable): fetch_queue's values.
__device__ inline void order_queue(const LocalArgs& g, int32_t d, int64_t built_n_total = -1,
                                   const DecHeader* built = nullptr, const QueueFetch* pre = nullptr) {
    __shared__ LocalLds s;
    const SnapLayout& L = g.L;
    const SnapView V = snap_view(const_cast<void*>(g.snap), L);
    int64_t n_total = built_n_total;
    if (built == nullptr) {
        const SnapHeader hdr = *V.hdr;
        if (!(hdr.magic == kSnapMagic && hdr.D == L.D && hdr.u_max == L.u_max && hdr.W == L.W)) {
            if (d == 0 && threadIdx.x == 0) raise_error(g.dev_err, MAPS_ERR_SNAPSHOT);
            return;
        }
        n_total = hdr.n_total;
    }
    const DecHeader h = built != nullptr ? *built : V.dec[d];
    if (!slice_ok(h, n_total, L)) {
        if (threadIdx.x == 0) raise_error(g.dev_err, MAPS_ERR_SNAPSHOT);
        return;
    }
    const QueueFetch f = pre != nullptr ? *pre : fetch_queue(g, d);
    const int64_t qlo = f.qlo, qhi = f.qhi;
    if (!(0 <= qlo && qlo <= qhi && qhi <= g.total)) {
        if (threadIdx.x == 0) { raise_error(g.dev_err, MAPS_ERR_SEG_OFFSETS); g.admitted[d] = 0; }
        return;
    }
    const int64_t n64 = qhi - qlo;
    if (n64 > kMaxQ) {
        if (threadIdx.x == 0) { raise_error(g.dev_err, MAPS_ERR_QUEUE_TOO_LONG); g.admitted[d] = 0; }
        return;
    }
    const int n = int(n64);
    const int32_t C = f.C;
    if (threadIdx.x == 0 && C < 0) raise_error(g.dev_err, MAPS_ERR_NEG_LEN);
    int n2 = 1;
    while (n2 < n) n2 <<= 1;

    if (n2 <= kWave) {
        // A queue of at most one wavefront: request i in lane i of every
        // wavefront.  Both orders by counting: the new position of i is the
        // number of requests before it by (class and key, index), its place
        // by bound the number before it by (bound, index), and the start of
        // its run of equal bounds the number with a smaller bound.  Wavefront
        // w counts against requests [4w, 4w + 4); wave 0 adds the counts.
        constexpr int kWaves = kOrderNT / kWave;
        constexpr int kPer = kWave / kWaves;   // requests each wavefront counts against
        const int i = int(threadIdx.x % kWave), w = int(threadIdx.x / kWave);
        bool neg = false;
        uint32_t h = ~0u, ue = ~0u;   // past the queue: after every request
        if (i < n) {
            neg = f.pr < 0;
            ue = uint32_t(f.u < 0 ? L.u_max : f.u);
            const bool promoted = g.qwait != nullptr && f.wait >= g.max_wait;
            h = promoted ? uint32_t(i) : (0x80000000u | ue);   // class bit, then index or bound
            if (w == 0) {
                s.pp[i] = f.pr < 0 ? 0 : f.pr;
                s.ue[i] = int32_t(ue);
            }
        }
        if (neg && w == 0) raise_error(g.dev_err, MAPS_ERR_NEG_LEN);
        uint32_t r1 = 0, r2 = 0, r3 = 0;
#pragma unroll
        for (int jj = 0; jj < kPer; ++jj) {
            const int j = w * kPer + jj;
            if (j >= n) break;   // uniform
            const uint32_t hj = __builtin_amdgcn_readlane(h, j), uj = __builtin_amdgcn_readlane(ue, j);
            r1 += (hj < h) | ((hj == h) & (j < i));
            r2 += (uj < ue) | ((uj == ue) & (j < i));
            r3 += uj < ue;
        }
        uint32_t* part = reinterpret_cast<uint32_t*>(s.keys);   // [3][kWaves][kWave], free until step 3
        part[(0 * kWaves + w) * kWave + i] = r1;
        part[(1 * kWaves + w) * kWave + i] = r2;
        part[(2 * kWaves + w) * kWave + i] = r3;
        __syncthreads();
        if (w == 0 && i < n) {
            uint32_t a1 = 0, a2 = 0, a3 = 0;
#pragma unroll
            for (int v = 0; v < kWaves; ++v) {
                a1 += part[(0 * kWaves + v) * kWave + i];
                a2 += part[(1 * kWaves + v) * kWave + i];
                a3 += part[(2 * kWaves + v) * kWave + i];
            }
            g.order[qlo + a1] = i;
            s.pos[i] = int32_t(a1);
            s.uidx[a2] = i;
            s.grp[a2] = int32_t(a3);
        }
        __syncthreads();
    } else {
        // 1. the new order (Eq. (7) with promotion)
        bool neg = false;
        for (int i = threadIdx.x; i < n2; i += kOrderNT) {
            if (i < n) {
                int32_t pr = g.qp[qlo + i], u = g.qU[qlo + i];
                neg |= pr < 0;
                s.pp[i] = pr < 0 ? 0 : pr;
                const int32_t ue = u < 0 ? L.u_max : u;
                s.ue[i] = ue;
                const bool promoted = g.qwait != nullptr && g.qwait[qlo + i] >= g.max_wait;
                const uint64_t cls = promoted ? 0ull : (1ull << 63);
                const uint64_t val = promoted ? uint64_t(i) : uint64_t(ue);
                s.keys[i] = cls | (val << 32) | uint64_t(uint32_t(i));
            } else {
                s.keys[i] = ~0ull;
            }
        }
        if (neg) raise_error(g.dev_err, MAPS_ERR_NEG_LEN);
        __syncthreads();
        bitonic_sort(s.keys, n2);
        for (int i = threadIdx.x; i < n; i += kOrderNT) {
            const int idx = int(uint32_t(s.keys[i]));
            g.order[qlo + i] = idx;
            s.pos[idx] = i;
        }
        __syncthreads();

        // 2. the queue sorted by bound
        for (int i = threadIdx.x; i < n2; i += kOrderNT)
            s.keys[i] = i < n ? ((uint64_t(uint32_t(s.ue[i])) << 32) | uint64_t(uint32_t(i))) : ~0ull;
        __syncthreads();
        bitonic_sort(s.keys, n2);
        for (int i = threadIdx.x; i < n; i += kOrderNT) s.uidx[i] = int(uint32_t(s.keys[i]));
        __syncthreads();
        block_scan<kOrderNT, true, false, false, int32_t>(
            n, 0,
            [&](int64_t i) { return (i == 0 || s.ue[s.uidx[i - 1]] != s.ue[s.uidx[i]]) ? int32_t(i) : 0; },
            [&](int64_t i, int32_t v) { s.grp[i] = v; }, s.red32);
    }

    // 3. admission: largest k with peak(k) <= C
    const uint2* rank = slice_rank(V, h);
    const int2* cold = slice_cold(V, h, L);
    int lo = 0;
    if (h.base_peak <= C) {
        int hi = n;
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            const int64_t pk = prefix_peak(s, n, mid, rank, cold, h.E, L.W);
            if (pk <= C) lo = mid; else hi = mid - 1;
        }
    }
    if (threadIdx.x == 0) g.admitted[d] = lo;
}

}  // namespace order
}  // namespace maps
