// Uncertainty-aware calibration (Sec. 3.2, Eqs. (2)-(4)) on gfx950.
//
// Per length bucket b the conformal quantile is the k_b-th smallest one-sided
// score s = max(0, L - L_hat), k_b = ceil((1 - alpha)(n_b + 1)) (infinite when
// k_b > n_b); every bound is then U = min(L_hat + q_b, u_max).
//
// Up to 1,024 buckets (and 8.4M residuals): a counting sort by bucket, then
// one workgroup per bucket selects.
//   cal_count         scores' buckets (binary search of the edges in LDS):
//                     per-workgroup bucket sizes and the largest score;
//   cal_offsets       per bucket: exclusive scan of the workgroups' sizes, the
//                     bucket size n_b, k_b, the largest score;
//   cal_scatter       each workgroup sorts its scores by bucket in LDS and
//                     writes every run to its place, bucket-major;
//   cal_bucket_select per bucket: most-significant-digit-first radix select
//                     of the k_b-th score over its run (kept in registers),
//                     8 bits a pass from the top digit of the largest score,
//                     histograms in LDS;
//   cal_apply         U = min(L_hat + q_b, u_max).
// More buckets: the same select over all buckets at once, one histogram
// pass and one selection kernel per 8-bit digit (cal_score, cal_rank,
// cal_hist, cal_select, cal_finish), histograms in LDS for up to 128 buckets.
// All reductions are integer additions, so the result is deterministic.
#include "maps_internal.hpp"

namespace maps {
namespace {

constexpr int kNT = 256;             // threads of the streaming kernels
constexpr int kApplyPer = 4;         // bounds per cal_apply thread (more waves beat more loads in flight)
constexpr int kHistNT = 1024;        // threads of the histogram kernel
constexpr int kLdsEdgesMax = 8192;   // buckets whose edges and sizes fit LDS
constexpr int kLdsHistBuckets = 128; // buckets whose 256-bin histograms fit LDS

struct CalWorkspace {
    int32_t* s;        // [n] scores
    uint16_t* b;       // [n] bucket ids
    uint32_t* cnt;     // [nb] bucket sizes
    int32_t* krem;     // [nb] rank still to find inside the prefix, -1 when q is infinite
    uint32_t* prefix;  // [nb] selected high digits of q
    uint32_t* hist;    // [nb][256]
    uint32_t* maxs;    // [1] largest score
    size_t bytes;
};

CalWorkspace cal_carve(void* base, int64_t n, int32_t nb) {
    CalWorkspace w;
    size_t off = 0;
    char* p = static_cast<char*>(base);
    auto take = [&](size_t bytes) { char* r = p ? p + off : nullptr; off += align256(bytes); return r; };
    w.s = reinterpret_cast<int32_t*>(take(size_t(n) * 4));
    w.b = reinterpret_cast<uint16_t*>(take(size_t(n) * 2));
    w.cnt = reinterpret_cast<uint32_t*>(take(size_t(nb) * 4));
    w.krem = reinterpret_cast<int32_t*>(take(size_t(nb) * 4));
    w.prefix = reinterpret_cast<uint32_t*>(take(size_t(nb) * 4));
    w.hist = reinterpret_cast<uint32_t*>(take(size_t(nb) * 256 * 4));
    w.maxs = reinterpret_cast<uint32_t*>(take(4));
    w.bytes = off;
    return w;
}

// Number of edges <= v among edges[0..ne-1] (upper bound of v).
__device__ inline int bucket_of(const int32_t* edges, int ne, int32_t v) {
    int lo = 0, hi = ne;
    while (lo < hi) {
        int mid = (lo + hi) >> 1;
        if (edges[mid] <= v) lo = mid + 1; else hi = mid;
    }
    return lo;
}

// bucket_of for kJ values at once, the searches interleaved (binary lifting
// over the sorted edges: the same count of edges <= v).
template <int kJ>
__device__ inline void buckets_of(const int32_t* edges, int ne, const int32_t (&v)[kJ], int (&b)[kJ]) {
    int step = 1;
    while (step * 2 <= ne) step *= 2;
#pragma unroll
    for (int j = 0; j < kJ; ++j) b[j] = 0;
    for (; step > 0; step >>= 1) {
#pragma unroll
        for (int j = 0; j < kJ; ++j) {
            const int np = b[j] + step;
            if (np <= ne && edges[np - 1] <= v[j]) b[j] = np;
        }
    }
}

__global__ void cal_init(int nb, uint32_t* cnt, uint32_t* hist, uint32_t* maxs) {
    const int64_t stride = int64_t(gridDim.x) * blockDim.x;
    for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < int64_t(nb) * 256; i += stride) {
        hist[i] = 0;
        if (i < nb) cnt[i] = 0;
        if (i == 0) maxs[0] = 0;
    }
}

template <bool kLds>
__global__ __launch_bounds__(kNT) void cal_score(const int32_t* __restrict__ pred,
                                                 const int32_t* __restrict__ truth, int64_t n,
                                                 const int32_t* __restrict__ edges, int nb,
                                                 int32_t* __restrict__ s_out, uint16_t* __restrict__ b_out,
                                                 uint32_t* __restrict__ cnt, uint32_t* __restrict__ maxs,
                                                 uint32_t* dev_err) {
    extern __shared__ int32_t lds[];
    const int ne = nb - 1;
    const int32_t* e = edges;
    uint32_t* c = cnt;
    if constexpr (kLds) {
        int32_t* le = lds;
        uint32_t* lc = reinterpret_cast<uint32_t*>(lds + ne);
        for (int i = threadIdx.x; i < ne; i += kNT) le[i] = edges[i];
        for (int i = threadIdx.x; i < nb; i += kNT) lc[i] = 0;
        __syncthreads();
        e = le;
        c = lc;
    }
    if (blockIdx.x == 0) {
        for (int i = threadIdx.x; i + 1 < ne; i += kNT)
            if (edges[i] > edges[i + 1]) raise_error(dev_err, MAPS_ERR_EDGES_UNSORTED);
    }
    uint32_t local_max = 0;
    bool bad = false;
    const int64_t stride = int64_t(gridDim.x) * kNT;
    for (int64_t i = int64_t(blockIdx.x) * kNT + threadIdx.x; i < n; i += stride) {
        int32_t p = pred[i], t = truth[i];
        bad |= (p < 0) | (t < 0);
        int64_t d = int64_t(t) - p;     // Eq. (2): s = max(0, L - L_hat)
        int32_t s = d <= 0 ? 0 : (d > INT32_MAX ? INT32_MAX : int32_t(d));
        int b = bucket_of(e, ne, p);
        s_out[i] = s;
        b_out[i] = uint16_t(b);
        atomicAdd(&c[b], 1u);
        local_max = local_max > uint32_t(s) ? local_max : uint32_t(s);
    }
    if (bad) raise_error(dev_err, MAPS_ERR_NEG_LEN);
    local_max = wave_reduce_max(local_max);
    if (threadIdx.x % kWave == 0 && local_max) atomicMax(maxs, local_max);
    if constexpr (kLds) {
        __syncthreads();
        for (int i = threadIdx.x; i < nb; i += kNT)
            if (c[i]) atomicAdd(&cnt[i], c[i]);
    }
}

__global__ void cal_rank(int nb, int32_t alpha_ppm, const uint32_t* cnt, int32_t* krem, uint32_t* prefix) {
    int b = blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= nb) return;
    int64_t nbk = cnt[b];
    int64_t k = ((int64_t(1000000 - alpha_ppm)) * (nbk + 1) + 999999) / 1000000;  // Eq. (3)
    krem[b] = (k <= nbk) ? int32_t(k) : -1;
    prefix[b] = 0;
}

__device__ inline bool pass_skipped(const uint32_t* maxs, int shift) {
    return shift > 0 && (maxs[0] >> shift) == 0u;
}

template <bool kLds>
__global__ __launch_bounds__(kHistNT) void cal_hist(const int32_t* __restrict__ s, const uint16_t* __restrict__ bk,
                                                    int64_t n, int nb, int shift,
                                                    const int32_t* __restrict__ krem,
                                                    const uint32_t* __restrict__ prefix,
                                                    uint32_t* __restrict__ hist, const uint32_t* maxs) {
    if (pass_skipped(maxs, shift)) return;
    extern __shared__ uint32_t lh[];
    uint32_t* h = hist;
    int32_t* lk = nullptr;
    uint32_t* lp = nullptr;
    if constexpr (kLds) {
        h = lh;
        lk = reinterpret_cast<int32_t*>(lh + nb * 256);
        lp = lh + nb * 256 + nb;
        for (int i = threadIdx.x; i < nb * 256; i += kHistNT) lh[i] = 0;
        for (int i = threadIdx.x; i < nb; i += kHistNT) { lk[i] = krem[i]; lp[i] = prefix[i]; }
        __syncthreads();
    }
    const int64_t stride = int64_t(gridDim.x) * kHistNT;
    for (int64_t i = int64_t(blockIdx.x) * kHistNT + threadIdx.x; i < n; i += stride) {
        int b = bk[i];
        int32_t k = kLds ? lk[b] : krem[b];
        if (k < 0) continue;
        uint32_t v = uint32_t(s[i]);
        uint32_t pre = kLds ? lp[b] : prefix[b];
        if (uint32_t(uint64_t(v) >> (shift + 8)) != pre) continue;
        atomicAdd(&h[b * 256 + ((v >> shift) & 255u)], 1u);
    }
    if constexpr (kLds) {
        __syncthreads();
        for (int i = threadIdx.x; i < nb * 256; i += kHistNT)
            if (lh[i]) atomicAdd(&hist[i], lh[i]);
    }
}

// One wavefront per bucket: the digit whose cumulative count reaches k.
__global__ __launch_bounds__(kNT) void cal_select(int nb, int shift, uint32_t* __restrict__ hist,
                                                  int32_t* __restrict__ krem, uint32_t* __restrict__ prefix,
                                                  const uint32_t* maxs) {
    if (pass_skipped(maxs, shift)) return;
    const int lane = threadIdx.x % kWave;
    const int b = blockIdx.x * (kNT / kWave) + threadIdx.x / kWave;
    if (b >= nb) return;
    uint32_t* row = hist + size_t(b) * 256;
    const int32_t k = krem[b];
    uint32_t h[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) { h[j] = row[lane * 4 + j]; row[lane * 4 + j] = 0; }
    if (k < 0) return;
    uint32_t mine = h[0] + h[1] + h[2] + h[3];
    uint32_t incl = wave_incl_scan_add(mine);
    uint32_t c = incl - mine;
    int digit = -1;
    uint32_t newk = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        if (digit < 0 && c < uint32_t(k) && c + h[j] >= uint32_t(k)) { digit = lane * 4 + j; newk = uint32_t(k) - c; }
        c += h[j];
    }
    uint64_t hit = __ballot(digit >= 0);
    if (hit == 0) return;  // cannot happen on consistent input
    int src = __ffsll((unsigned long long)hit) - 1;
    digit = __shfl(digit, src, kWave);
    newk = __shfl(newk, src, kWave);
    if (lane == 0) {
        prefix[b] = (prefix[b] << 8) | uint32_t(digit);
        krem[b] = int32_t(newk);
    }
}

__global__ void cal_finish(int nb, const int32_t* krem, const uint32_t* prefix, const uint32_t* cnt,
                           int32_t* q_out, int32_t* count_out) {
    int b = blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= nb) return;
    q_out[b] = krem[b] < 0 ? MAPS_Q_INF : int32_t(prefix[b]);
    count_out[b] = int32_t(cnt[b]);
}

template <bool kLds>
__global__ __launch_bounds__(kNT) void cal_apply(const int32_t* __restrict__ pred, int64_t m,
                                                 const int32_t* __restrict__ edges, int nb,
                                                 const int32_t* __restrict__ q, int32_t u_max,
                                                 int32_t* __restrict__ U) {
    extern __shared__ int32_t lds[];
    const int ne = nb - 1;
    const int32_t* e = edges;
    const int32_t* qq = q;
    if constexpr (kLds) {
        int32_t* le = lds;
        int32_t* lq = lds + ne;
        for (int i = threadIdx.x; i < ne; i += kNT) le[i] = edges[i];
        for (int i = threadIdx.x; i < nb; i += kNT) lq[i] = q[i];
        __syncthreads();
        e = le;
        qq = lq;
    }
    constexpr int kA = kApplyPer;   // predictions per thread in flight
    const int64_t stride = int64_t(gridDim.x) * kNT * kA;
    for (int64_t c0 = int64_t(blockIdx.x) * kNT * kA; c0 < m; c0 += stride) {
        int32_t p[kA];
        int b[kA];
#pragma unroll
        for (int j = 0; j < kA; ++j) {
            const int64_t i = c0 + int64_t(j) * kNT + threadIdx.x;
            p[j] = i < m ? pred[i] : -1;
        }
        buckets_of<kA>(e, ne, p, b);
#pragma unroll
        for (int j = 0; j < kA; ++j) {
            const int64_t i = c0 + int64_t(j) * kNT + threadIdx.x;
            if (i >= m) continue;
            int32_t out = -1;   // no prediction: no bound
            if (p[j] >= 0) {
                const int32_t qb = qq[b[j]];
                const int64_t v = int64_t(p[j]) + qb;   // Eq. (4)
                out = (qb == MAPS_Q_INF || v > u_max) ? u_max : int32_t(v);
            }
            U[i] = out;
        }
    }
}

// ---------------------------------------------------------------------------
// Counting-sort path (nb <= kFastBuckets)
// ---------------------------------------------------------------------------
constexpr int kFastBuckets = 1024;
constexpr int kSortNT = 256;
constexpr int kJ = 4;                                   // residuals per thread
constexpr int64_t kPerBlock = int64_t(kSortNT) * kJ;    // residuals per workgroup of cal_count / cal_scatter
constexpr int64_t kSortMaxBlocks = 4096;                // larger sets take the all-bucket path
constexpr int kSelNT = 1024;
constexpr int kKeep = 24;   // scores per thread the bucket select keeps in registers across passes

int64_t sort_blocks(int64_t n) { return (n + kPerBlock - 1) / kPerBlock; }

struct FastWorkspace {
    uint32_t* cnt_part;   // [nb][blocks] bucket sizes of each workgroup
    uint32_t* off_part;   // [nb][blocks] where each workgroup's run starts inside the bucket
    uint32_t* max_part;   // [blocks] largest score of each workgroup
    uint32_t* bcount;     // [nb] bucket sizes
    uint32_t* bmax;       // [nb] largest score (the same for every bucket)
    int32_t* krank;       // [nb] k_b, -1 when the quantile is infinite
    int32_t* sorted;      // [n] scores, bucket-major
    size_t bytes;
};

FastWorkspace fast_carve(void* base, int64_t n, int32_t nb) {
    const int64_t blocks = sort_blocks(n);
    FastWorkspace w;
    size_t off = 0;
    char* p = static_cast<char*>(base);
    auto take = [&](size_t bytes) { char* r = p ? p + off : nullptr; off += align256(bytes); return r; };
    w.cnt_part = reinterpret_cast<uint32_t*>(take(size_t(blocks) * nb * 4));
    w.off_part = reinterpret_cast<uint32_t*>(take(size_t(blocks) * nb * 4));
    w.max_part = reinterpret_cast<uint32_t*>(take(size_t(blocks) * 4));
    w.bcount = reinterpret_cast<uint32_t*>(take(size_t(nb) * 4));
    w.bmax = reinterpret_cast<uint32_t*>(take(size_t(nb) * 4));
    w.krank = reinterpret_cast<int32_t*>(take(size_t(nb) * 4));
    w.sorted = reinterpret_cast<int32_t*>(take(size_t(n) * 4));
    w.bytes = off;
    return w;
}

bool fast_path(int64_t n, int32_t nb) { return nb <= kFastBuckets && sort_blocks(n) <= kSortMaxBlocks; }

// Score of one residual (Eq. (2)): max(0, L - L_hat), saturated at INT32_MAX.
__device__ inline int32_t score_of(int32_t p, int32_t t) {
    const int64_t d = int64_t(t) - p;
    return d <= 0 ? 0 : (d > INT32_MAX ? INT32_MAX : int32_t(d));
}

// The kJ residuals of this thread in workgroup blockIdx.x: prompt
// prediction, score, bucket; `valid` masks the ones past n.
struct Residuals {
    int32_t p[kJ], s[kJ];
    int b[kJ];
    bool valid[kJ];
};

__device__ inline void load_residuals(const int32_t* __restrict__ pred, const int32_t* __restrict__ truth, int64_t n,
                                      const int32_t* le, int ne, Residuals& r, bool& bad) {
    const int64_t lo = int64_t(blockIdx.x) * kPerBlock;
    int32_t t[kJ];
#pragma unroll
    for (int j = 0; j < kJ; ++j) {
        const int64_t i = lo + int64_t(j) * kSortNT + threadIdx.x;
        r.valid[j] = i < n;
        r.p[j] = r.valid[j] ? pred[i] : 0;
        t[j] = r.valid[j] ? truth[i] : 0;
    }
    buckets_of<kJ>(le, ne, r.p, r.b);
#pragma unroll
    for (int j = 0; j < kJ; ++j) {
        bad |= r.valid[j] & ((r.p[j] < 0) | (t[j] < 0));
        r.s[j] = score_of(r.p[j], t[j]);
    }
}

__global__ __launch_bounds__(kSortNT) void cal_count(const int32_t* __restrict__ pred,
                                                     const int32_t* __restrict__ truth, int64_t n,
                                                     const int32_t* __restrict__ edges, int nb, int64_t blocks,
                                                     uint32_t* __restrict__ cnt_part, uint32_t* __restrict__ max_part,
                                                     uint32_t* dev_err) {
    extern __shared__ int32_t lds[];
    __shared__ uint32_t red[kSortNT / kWave];
    const int ne = nb - 1;
    int32_t* le = lds;
    uint32_t* lc = reinterpret_cast<uint32_t*>(lds + ne);
    for (int i = threadIdx.x; i < ne; i += kSortNT) le[i] = edges[i];
    for (int i = threadIdx.x; i < nb; i += kSortNT) lc[i] = 0;
    if (blockIdx.x == 0)
        for (int i = threadIdx.x; i + 1 < ne; i += kSortNT)
            if (edges[i] > edges[i + 1]) raise_error(dev_err, MAPS_ERR_EDGES_UNSORTED);
    __syncthreads();
    Residuals r;
    bool bad = false;
    load_residuals(pred, truth, n, le, ne, r, bad);
    uint32_t mx = 0;
#pragma unroll
    for (int j = 0; j < kJ; ++j) {
        if (!r.valid[j]) continue;
        atomicAdd(&lc[r.b[j]], 1u);
        mx = mx > uint32_t(r.s[j]) ? mx : uint32_t(r.s[j]);
    }
    if (bad) raise_error(dev_err, MAPS_ERR_NEG_LEN);
    mx = block_reduce_max<kSortNT>(mx, red);   // starts with a barrier: the counts are complete
    for (int b = threadIdx.x; b < nb; b += kSortNT) cnt_part[int64_t(b) * blocks + blockIdx.x] = lc[b];
    if (threadIdx.x == 0) max_part[blockIdx.x] = mx;
}

__global__ __launch_bounds__(kSortNT) void cal_offsets(int nb, int64_t blocks, int32_t alpha_ppm,
                                                       const uint32_t* __restrict__ cnt_part,
                                                       const uint32_t* __restrict__ max_part,
                                                       uint32_t* __restrict__ off_part, uint32_t* __restrict__ bcount,
                                                       uint32_t* __restrict__ bmax, int32_t* __restrict__ krank) {
    __shared__ uint32_t tmp[kSortNT / kWave];
    const int b = blockIdx.x;
    const uint32_t* col = cnt_part + int64_t(b) * blocks;
    uint32_t* ocol = off_part + int64_t(b) * blocks;
    const uint32_t total = block_scan<kSortNT, false, false, true, uint32_t>(
        blocks, 0u, [&](int64_t i) { return col[i]; }, [&](int64_t i, uint32_t v) { ocol[i] = v; }, tmp);
    uint32_t mx = 0;
    for (int64_t i = threadIdx.x; i < blocks; i += kSortNT) mx = mx > max_part[i] ? mx : max_part[i];
    mx = block_reduce_max<kSortNT>(mx, tmp);
    if (threadIdx.x == 0) {
        const int64_t nbk = total;
        const int64_t k = (int64_t(1000000 - alpha_ppm) * (nbk + 1) + 999999) / 1000000;  // Eq. (3)
        bcount[b] = total;
        bmax[b] = mx;
        krank[b] = k <= nbk ? int32_t(k) : -1;
    }
}

// Each workgroup sorts its residuals' scores by bucket in LDS, then writes
// every bucket's run to its place in the bucket-major array (consecutive
// scores of a run go to consecutive addresses).
__global__ __launch_bounds__(kSortNT) void cal_scatter(const int32_t* __restrict__ pred,
                                                       const int32_t* __restrict__ truth, int64_t n,
                                                       const int32_t* __restrict__ edges, int nb, int64_t blocks,
                                                       const uint32_t* __restrict__ bcount,
                                                       const uint32_t* __restrict__ off_part,
                                                       int32_t* __restrict__ sorted) {
    extern __shared__ int32_t lds[];
    __shared__ uint32_t tmp[kSortNT / kWave];
    const int ne = nb - 1;
    int32_t* le = lds;                                              // [ne]
    uint32_t* lcnt = reinterpret_cast<uint32_t*>(le + ne);          // [nb] local sizes, then local starts
    uint32_t* gdst = lcnt + nb;                                     // [nb] global start of the local run
    int32_t* lsort = reinterpret_cast<int32_t*>(gdst + nb);         // [kPerBlock] scores by bucket
    uint16_t* lbkt = reinterpret_cast<uint16_t*>(lsort + kPerBlock);   // [kPerBlock] their buckets
    for (int i = threadIdx.x; i < ne; i += kSortNT) le[i] = edges[i];
    for (int i = threadIdx.x; i < nb; i += kSortNT) lcnt[i] = 0;
    // start of each bucket's run in the bucket-major array
    block_scan<kSortNT, false, false, true, uint32_t>(
        nb, 0u, [&](int64_t i) { return bcount[i]; }, [&](int64_t i, uint32_t v) { gdst[i] = v; }, tmp);
    for (int b = threadIdx.x; b < nb; b += kSortNT) gdst[b] += off_part[int64_t(b) * blocks + blockIdx.x];
    Residuals r;
    bool bad = false;
    load_residuals(pred, truth, n, le, ne, r, bad);
    uint32_t rank[kJ];
#pragma unroll
    for (int j = 0; j < kJ; ++j) rank[j] = r.valid[j] ? atomicAdd(&lcnt[r.b[j]], 1u) : 0u;
    __syncthreads();
    block_scan<kSortNT, false, false, true, uint32_t>(
        nb, 0u, [&](int64_t i) { return lcnt[i]; }, [&](int64_t i, uint32_t v) { lcnt[i] = v; }, tmp);
#pragma unroll
    for (int j = 0; j < kJ; ++j) {
        if (!r.valid[j]) continue;
        const uint32_t at = lcnt[r.b[j]] + rank[j];
        lsort[at] = r.s[j];
        lbkt[at] = uint16_t(r.b[j]);
    }
    __syncthreads();
    const int64_t lo = int64_t(blockIdx.x) * kPerBlock;
    const int cnt = int(n - lo < kPerBlock ? n - lo : kPerBlock);
    for (int i = threadIdx.x; i < cnt; i += kSortNT) {
        const int b = lbkt[i];
        const uint32_t pos = gdst[b] + uint32_t(i) - lcnt[b];
        if (pos < uint64_t(n)) sorted[pos] = lsort[i];   // always: the runs partition [0, n)
    }
}

// Digit of the k-th element among the 256 bins of hist (one wavefront).
__device__ inline void pick_digit(const uint32_t* hist, int32_t k, uint32_t* pick) {
    const int lane = threadIdx.x;
    uint32_t h[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) h[j] = hist[lane * 4 + j];
    const uint32_t mine = h[0] + h[1] + h[2] + h[3];
    uint32_t c = wave_incl_scan_add(mine) - mine;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        if (c < uint32_t(k) && c + h[j] >= uint32_t(k)) { pick[0] = uint32_t(lane * 4 + j); pick[1] = uint32_t(k) - c; }
        c += h[j];
    }
}

// Histogram update of one score's digit; the lanes holding the first active
// lane's digit add it with one atomic.
__device__ inline void hist_add(uint32_t* hist, uint32_t digit) {
    const uint32_t lead = __builtin_amdgcn_readfirstlane(digit);
    const uint64_t same = __ballot(digit == lead);
    if (digit != lead) atomicAdd(&hist[digit], 1u);
    else if (int(threadIdx.x % kWave) == __ffsll((unsigned long long)same) - 1)
        atomicAdd(&hist[lead], uint32_t(__popcll(same)));
}

// One workgroup per bucket: the k_b-th smallest score of its run, most
// significant 8-bit digit first from the top digit of the largest score.  A
// run of at most kSelNT * kKeep scores stays in registers across passes.
__global__ __launch_bounds__(kSelNT) void cal_bucket_select(int nb, const int32_t* __restrict__ sorted,
                                                            const uint32_t* __restrict__ bcount,
                                                            const uint32_t* __restrict__ bmax,
                                                            const int32_t* __restrict__ krank,
                                                            int32_t* __restrict__ q_out,
                                                            int32_t* __restrict__ count_out) {
    __shared__ uint32_t hist[256];
    __shared__ uint32_t red[kSelNT / kWave];
    __shared__ uint32_t pick[2];
    const int b = blockIdx.x;
    uint32_t before = 0;
    for (int i = threadIdx.x; i < b; i += kSelNT) before += bcount[i];
    const uint32_t base = block_reduce_add<kSelNT>(before, red);
    const uint32_t nbk = bcount[b];
    int32_t k = krank[b];
    if (threadIdx.x == 0) count_out[b] = int32_t(nbk);
    if (k < 0) {
        if (threadIdx.x == 0) q_out[b] = MAPS_Q_INF;
        return;
    }
    const uint32_t mx = bmax[b];
    const int top = mx >> 24 ? 24 : (mx >> 16 ? 16 : (mx >> 8 ? 8 : 0));
    const int32_t* v = sorted + base;
    const bool in_regs = nbk <= uint32_t(kSelNT) * kKeep;
    uint32_t x[kKeep];
    if (in_regs) {
#pragma unroll
        for (int j = 0; j < kKeep; ++j) {
            const uint32_t i = uint32_t(j) * kSelNT + threadIdx.x;
            x[j] = i < nbk ? uint32_t(v[i]) : 0u;
        }
    }
    uint32_t prefix = 0;
    for (int shift = top; shift >= 0; shift -= 8) {
        if (threadIdx.x < 256) hist[threadIdx.x] = 0;
        __syncthreads();
        if (in_regs) {
#pragma unroll
            for (int j = 0; j < kKeep; ++j) {
                const uint32_t i = uint32_t(j) * kSelNT + threadIdx.x;
                const uint32_t y = x[j] >> shift;
                if (i < nbk && (y >> 8) == prefix) hist_add(hist, y & 255u);
            }
        } else {
            for (uint32_t c0 = 0; c0 < nbk; c0 += kSelNT * kJ) {
                uint32_t y[kJ];
#pragma unroll
                for (int j = 0; j < kJ; ++j) {
                    const uint32_t i = c0 + uint32_t(j) * kSelNT + threadIdx.x;
                    y[j] = i < nbk ? uint32_t(v[i]) >> shift : 0u;
                }
#pragma unroll
                for (int j = 0; j < kJ; ++j) {
                    const uint32_t i = c0 + uint32_t(j) * kSelNT + threadIdx.x;
                    if (i < nbk && (y[j] >> 8) == prefix) hist_add(hist, y[j] & 255u);
                }
            }
        }
        __syncthreads();
        if (threadIdx.x < kWave) pick_digit(hist, k, pick);
        __syncthreads();
        prefix = (prefix << 8) | pick[0];
        k = int32_t(pick[1]);
        __syncthreads();
    }
    if (threadIdx.x == 0) q_out[b] = int32_t(prefix);
}

int grid_for(int64_t n, int nt, int per_thread, int cap) {
    int64_t g = (n + int64_t(nt) * per_thread - 1) / (int64_t(nt) * per_thread);
    if (g < 1) g = 1;
    if (g > cap) g = cap;
    return int(g);
}

}  // namespace
}  // namespace maps

using namespace maps;

extern "C" size_t maps_calibrate_workspace_size(int64_t n, int32_t nb) {
    if (n < 0 || nb < 1) return 0;
    return fast_path(n, nb) ? fast_carve(nullptr, n, nb).bytes : cal_carve(nullptr, n, nb).bytes;
}

namespace {

// Calibration by counting sort (up to kFastBuckets buckets and
// kSortMaxBlocks * kPerBlock residuals), then one workgroup per bucket.
maps_status calibrate_fast(const int32_t* pred, const int32_t* truth, int64_t n, const int32_t* edges, int32_t nb,
                           int32_t alpha_ppm, int32_t* q_out, int32_t* count_out, uint32_t* dev_err,
                           void* workspace, hipStream_t stream) {
    const FastWorkspace w = fast_carve(workspace, n, nb);
    const int64_t blocks = sort_blocks(n);
    const size_t lds_count = size_t(2 * nb) * 4;   // edges and per-bucket counters
    const size_t lds_scatter = size_t(3 * nb) * 4 + size_t(kPerBlock) * 6;
    if (n > 0) {
        hipLaunchKernelGGL(cal_count, dim3(unsigned(blocks)), dim3(kSortNT), lds_count, stream, pred, truth, n,
                           edges, nb, blocks, w.cnt_part, w.max_part, dev_err);
        MAPS_CHECK_LAUNCH();
    }
    hipLaunchKernelGGL(cal_offsets, dim3(unsigned(nb)), dim3(kSortNT), 0, stream, nb, blocks, alpha_ppm,
                       w.cnt_part, w.max_part, w.off_part, w.bcount, w.bmax, w.krank);
    MAPS_CHECK_LAUNCH();
    if (n > 0) {
        hipLaunchKernelGGL(cal_scatter, dim3(unsigned(blocks)), dim3(kSortNT), lds_scatter, stream, pred, truth, n,
                           edges, nb, blocks, w.bcount, w.off_part, w.sorted);
        MAPS_CHECK_LAUNCH();
    }
    hipLaunchKernelGGL(cal_bucket_select, dim3(unsigned(nb)), dim3(kSelNT), 0, stream, nb, w.sorted, w.bcount,
                       w.bmax, w.krank, q_out, count_out);
    MAPS_CHECK_LAUNCH();
    return MAPS_OK;
}

maps_status calibrate_general(const int32_t* pred, const int32_t* truth, int64_t n, const int32_t* edges,
                              int32_t nb, int32_t alpha_ppm, int32_t* q_out, int32_t* count_out, uint32_t* dev_err,
                              void* workspace, hipStream_t stream) {
    CalWorkspace w = cal_carve(workspace, n, nb);

    const bool lds_edges = nb <= kLdsEdgesMax;
    const bool lds_hist = nb <= kLdsHistBuckets;
    const int ne = nb - 1;

    hipLaunchKernelGGL(cal_init, dim3(grid_for(int64_t(nb) * 256, kNT, 1, 1024)), dim3(kNT), 0, stream,
                       nb, w.cnt, w.hist, w.maxs);
    MAPS_CHECK_LAUNCH();
    if (n > 0) {
        const int g = grid_for(n, kNT, 16, 2048);
        if (lds_edges)
            hipLaunchKernelGGL(cal_score<true>, dim3(g), dim3(kNT), size_t(ne + nb) * 4, stream,
                               pred, truth, n, edges, nb, w.s, w.b, w.cnt, w.maxs, dev_err);
        else
            hipLaunchKernelGGL(cal_score<false>, dim3(g), dim3(kNT), 0, stream,
                               pred, truth, n, edges, nb, w.s, w.b, w.cnt, w.maxs, dev_err);
        MAPS_CHECK_LAUNCH();
    }
    hipLaunchKernelGGL(cal_rank, dim3((nb + kNT - 1) / kNT), dim3(kNT), 0, stream,
                       nb, alpha_ppm, w.cnt, w.krem, w.prefix);
    MAPS_CHECK_LAUNCH();
    if (n > 0) {
        const int gh = grid_for(n, kHistNT, 16, 256);
        for (int shift = 24; shift >= 0; shift -= 8) {
            if (lds_hist) {
                allow_dynamic_lds(cal_hist<true>, size_t(nb) * (256 + 2) * 4);
                hipLaunchKernelGGL(cal_hist<true>, dim3(gh), dim3(kHistNT), size_t(nb) * (256 + 2) * 4, stream,
                                   w.s, w.b, n, nb, shift, w.krem, w.prefix, w.hist, w.maxs);
            } else {
                hipLaunchKernelGGL(cal_hist<false>, dim3(gh), dim3(kHistNT), 0, stream,
                                   w.s, w.b, n, nb, shift, w.krem, w.prefix, w.hist, w.maxs);
            }
            MAPS_CHECK_LAUNCH();
            hipLaunchKernelGGL(cal_select, dim3((nb + kNT / kWave - 1) / (kNT / kWave)), dim3(kNT), 0, stream,
                               nb, shift, w.hist, w.krem, w.prefix, w.maxs);
            MAPS_CHECK_LAUNCH();
        }
    }
    hipLaunchKernelGGL(cal_finish, dim3((nb + kNT - 1) / kNT), dim3(kNT), 0, stream,
                       nb, w.krem, w.prefix, w.cnt, q_out, count_out);
    MAPS_CHECK_LAUNCH();
    return MAPS_OK;
}

}  // namespace

extern "C" maps_status maps_calibrate(const int32_t* pred, const int32_t* truth, int64_t n,
                                      const int32_t* edges, int32_t nb, int32_t alpha_ppm,
                                      int32_t* q_out, int32_t* count_out,
                                      const int32_t* apply_pred, int64_t m, int32_t u_max, int32_t* U_out,
                                      uint32_t* dev_err, void* workspace, size_t workspace_bytes,
                                      hipStream_t stream) {
    if (n < 0 || m < 0 || nb < 1 || nb > 65536 || u_max < 0) return MAPS_E_SIZE;
    if (alpha_ppm <= 0 || alpha_ppm >= 1000000) return MAPS_E_ALPHA;
    if (!q_out || !count_out || !dev_err || (n > 0 && (!pred || !truth)) || (nb > 1 && !edges) ||
        (m > 0 && (!apply_pred || !U_out)) || !workspace)
        return MAPS_E_NULL;
    if (workspace_bytes < maps_calibrate_workspace_size(n, nb)) return MAPS_E_WORKSPACE;
    const int ne = nb - 1;
    if (fast_path(n, nb)) {
        const maps_status st =
            calibrate_fast(pred, truth, n, edges, nb, alpha_ppm, q_out, count_out, dev_err, workspace, stream);
        if (st != MAPS_OK) return st;
    } else {
        const maps_status st =
            calibrate_general(pred, truth, n, edges, nb, alpha_ppm, q_out, count_out, dev_err, workspace, stream);
        if (st != MAPS_OK) return st;
    }
    if (m > 0) {
        const bool lds_edges = nb <= kLdsEdgesMax;
        const int g = grid_for(m, kNT, kApplyPer, 8192);
        if (lds_edges)
            hipLaunchKernelGGL(cal_apply<true>, dim3(g), dim3(kNT), size_t(ne + nb) * 4, stream,
                               apply_pred, m, edges, nb, q_out, u_max, U_out);
        else
            hipLaunchKernelGGL(cal_apply<false>, dim3(g), dim3(kNT), 0, stream,
                               apply_pred, m, edges, nb, q_out, u_max, U_out);
        MAPS_CHECK_LAUNCH();
    }
    return MAPS_OK;
}


