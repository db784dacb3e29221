// Uncertainty-aware calibration (Sec. 3.2, Eqs. (2)-(4)) on gfx950.
//
// Per length bucket b the conformal quantile is the k_b-th smallest one-sided
// score s = max(0, L - L_hat), k_b = ceil((1 - alpha)(n_b + 1)) (infinite when
// k_b > n_b); every bound is then U = min(L_hat + q_b, u_max).
//
// Up to 1,024 buckets (and 4.2M residuals): chunks sorted by bucket, then one
// workgroup per bucket selects.
//   cal_chunk_sort    per chunk of 4,096 residuals: scores and buckets (binary
//                     search of the edges in LDS), a counting sort of the
//                     chunk by bucket in LDS written back contiguously, the
//                     size and start of every bucket's run in the chunk, the
//                     chunk's largest score;
//   cal_bucket_select per bucket: n_b and k_b from its runs' sizes, its runs
//                     gathered into LDS and registers, then a most-
//                     significant-digit-first radix select of the k_b-th
//                     score, 8 bits a pass from the top digit of the largest
//                     score, histograms in LDS;
//   cal_apply         U = min(L_hat + q_b, u_max).
// More buckets or residuals: the same select over all buckets at once, one histogram
// pass and one selection kernel per 8-bit digit (cal_score, cal_rank,
// cal_hist, cal_select, cal_finish), histograms in LDS for up to 128 buckets.
// All reductions are integer additions, so the result is deterministic.
#include <cstdlib>
#include <mutex>
#include <unordered_map>

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
constexpr int kSortNT = 1024;
constexpr int kJ = 4;                                  // residuals per thread
constexpr int64_t kChunk = int64_t(kSortNT) * kJ;      // residuals per workgroup of cal_chunk_sort
constexpr int64_t kSortMaxChunks = 1024;               // larger sets take the all-bucket path
constexpr int kSelNT = 1024;
constexpr int kSelWaves = kSelNT / kWave;
constexpr int kKeep = 24;         // scores per thread the bucket select keeps in registers across passes
constexpr int kGatherRuns = 16;   // runs a wavefront of the select loads at once
constexpr size_t kSelStageBytes = size_t(kSelNT) * kKeep * 4;
static_assert(kSortMaxChunks <= kSelNT, "the select holds one run of its bucket per thread");
static_assert(kKeep % 4 == 0 && kGatherRuns <= kWave, "select slots come in groups of four");

int64_t sort_chunks(int64_t n) { return (n + kChunk - 1) / kChunk; }

struct FastWorkspace {
    uint32_t* run_cnt;     // [nb][chunks] scores of bucket b in chunk c (the run of b in c)
    uint32_t* run_start;   // [nb][chunks] where that run starts inside its chunk
    uint32_t* max_part;    // [chunks] largest score of each chunk
    int32_t* sorted;       // [n] scores, every chunk of kChunk sorted by bucket
    uint64_t* qflag;       // [nb] 1 << 32 | q_b once bucket b is selected (the fused apply waits on them)
    size_t bytes;
};

FastWorkspace fast_carve(void* base, int64_t n, int32_t nb) {
    const int64_t chunks = sort_chunks(n);
    FastWorkspace w;
    size_t off = 0;
    char* p = static_cast<char*>(base);
    auto take = [&](size_t bytes) { char* r = p ? p + off : nullptr; off += align256(bytes); return r; };
    w.run_cnt = reinterpret_cast<uint32_t*>(take(size_t(chunks) * nb * 4));
    w.run_start = reinterpret_cast<uint32_t*>(take(size_t(chunks) * nb * 4));
    w.max_part = reinterpret_cast<uint32_t*>(take(size_t(chunks) * 4));
    w.sorted = reinterpret_cast<int32_t*>(take(size_t(n) * 4));
    w.qflag = reinterpret_cast<uint64_t*>(take(size_t(nb) * 8));
    w.bytes = off;
    return w;
}

bool fast_path(int64_t n, int32_t nb) { return nb <= kFastBuckets && sort_chunks(n) <= kSortMaxChunks; }

// Score of one residual (Eq. (2)): max(0, L - L_hat), saturated at INT32_MAX.
__device__ inline int32_t score_of(int32_t p, int32_t t) {
    const int64_t d = int64_t(t) - p;
    return d <= 0 ? 0 : (d > INT32_MAX ? INT32_MAX : int32_t(d));
}

// The kJ residuals of this thread in chunk blockIdx.x: prompt prediction,
// score, bucket; `valid` masks the ones past n.
struct Residuals {
    int32_t p[kJ], s[kJ];
    int b[kJ];
    bool valid[kJ];
};

// Loads only: issued before the workgroup stages its tables, so that both
// latencies overlap.
__device__ inline void fetch_residuals(const int32_t* __restrict__ pred, const int32_t* __restrict__ truth,
                                       int64_t n, Residuals& r) {
    const int64_t lo = int64_t(blockIdx.x) * kChunk;
#pragma unroll
    for (int j = 0; j < kJ; ++j) {
        const int64_t i = lo + int64_t(j) * kSortNT + threadIdx.x;
        r.valid[j] = i < n;
        r.p[j] = r.valid[j] ? pred[i] : 0;
        r.s[j] = r.valid[j] ? truth[i] : 0;   // the true length until classify_residuals
    }
}

__device__ inline void classify_residuals(const int32_t* le, int ne, Residuals& r, bool& bad) {
    buckets_of<kJ>(le, ne, r.p, r.b);
#pragma unroll
    for (int j = 0; j < kJ; ++j) {
        bad |= r.valid[j] & ((r.p[j] < 0) | (r.s[j] < 0));
        r.s[j] = score_of(r.p[j], r.s[j]);
    }
}

// One workgroup per chunk of kChunk residuals: scores and buckets, then a
// counting sort of the chunk by bucket in LDS, written back in place of the
// chunk (one 16-byte store a thread); the size and start of every bucket's
// run in the chunk, bucket-major; the chunk's largest score.
__global__ __launch_bounds__(kSortNT) void cal_chunk_sort(const int32_t* __restrict__ pred,
                                                          const int32_t* __restrict__ truth, int64_t n,
                                                          const int32_t* __restrict__ edges, int nb, int64_t chunks,
                                                          uint32_t* __restrict__ run_cnt,
                                                          uint32_t* __restrict__ run_start,
                                                          uint32_t* __restrict__ max_part,
                                                          int32_t* __restrict__ sorted, uint64_t* qflag,
                                                          uint32_t* dev_err) {
    extern __shared__ __align__(16) int32_t chunk_lds[];
    __shared__ uint32_t red[kSortNT / kWave];
    Residuals r;
    fetch_residuals(pred, truth, n, r);
    const int ne = nb - 1;
    int32_t* lsort = chunk_lds;                                            // [kChunk] scores by bucket
    int32_t* le = lsort + kChunk;                                    // [ne]
    uint32_t* lcnt = reinterpret_cast<uint32_t*>(le + ne);           // [nb] run sizes
    uint32_t* lstart = lcnt + nb;                                    // [nb] run starts
    for (int i = threadIdx.x; i < ne; i += kSortNT) le[i] = edges[i];
    for (int i = threadIdx.x; i < nb; i += kSortNT) lcnt[i] = 0;
    if (blockIdx.x == 0)
        for (int i = threadIdx.x; i + 1 < ne; i += kSortNT)
            if (edges[i] > edges[i + 1]) raise_error(dev_err, MAPS_ERR_EDGES_UNSORTED);
    __syncthreads();
    bool bad = false;
    classify_residuals(le, ne, r, bad);
    uint32_t rank[kJ];
    uint32_t mx = 0;
#pragma unroll
    for (int j = 0; j < kJ; ++j) {
        rank[j] = r.valid[j] ? atomicAdd(&lcnt[r.b[j]], 1u) : 0u;
        if (r.valid[j]) mx = mx > uint32_t(r.s[j]) ? mx : uint32_t(r.s[j]);
    }
    if (bad) raise_error(dev_err, MAPS_ERR_NEG_LEN);
    mx = block_reduce_max<kSortNT>(mx, red);   // starts with a barrier: the run sizes are complete
    const int64_t c = blockIdx.x;
    block_scan<kSortNT, false, false, true, uint32_t>(
        nb, 0u, [&](int64_t i) { return lcnt[i]; }, [&](int64_t i, uint32_t v) { lstart[i] = v; },
        red);   // ends with a barrier: the run starts are complete
#pragma unroll
    for (int j = 0; j < kJ; ++j)
        if (r.valid[j]) lsort[lstart[r.b[j]] + rank[j]] = r.s[j];
    __syncthreads();
    // global stores only after the last barrier (a barrier waits for every
    // store in flight)
    for (int i = threadIdx.x; i < nb; i += kSortNT) {
        run_cnt[int64_t(i) * chunks + c] = lcnt[i];
        run_start[int64_t(i) * chunks + c] = lstart[i];
    }
    const int64_t lo = c * kChunk;
    const int cnt = int(n - lo < kChunk ? n - lo : kChunk);
    if (cnt == kChunk) {
        reinterpret_cast<int4*>(sorted + lo)[threadIdx.x] = reinterpret_cast<const int4*>(lsort)[threadIdx.x];
    } else {
        for (int i = threadIdx.x; i < cnt; i += kSortNT) sorted[lo + i] = lsort[i];
    }
    if (threadIdx.x == 0) max_part[c] = mx;
    if (c == 0)   // the selection that follows raises them
        for (int i = threadIdx.x; i < nb; i += kSortNT) qflag[i] = 0u;
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

// Histogram update of one score's digit when `take`.  Digit 0 is the common
// one (every score of zero, and short scores on the top digit): those lanes
// are counted by a ballot into the wavefront-uniform `zeros`, which the
// caller adds to bin 0 once; the other lanes add one each.  Called by whole
// wavefronts.
__device__ inline void hist_add(uint32_t* hist, bool take, uint32_t digit, uint32_t& zeros) {
    zeros += uint32_t(__popcll(__ballot(take && digit == 0)));
    if (take && digit != 0) atomicAdd(&hist[digit], 1u);
}

__device__ inline void hist_flush_zeros(uint32_t* hist, uint32_t zeros) {
    if ((threadIdx.x % kWave) == 0 && zeros != 0) atomicAdd(&hist[0], zeros);
}

// Thread 0 of a selecting workgroup: bucket b's quantile, published with
// its ready bit in one device-coherent word (the value is the flag, so no
// fence orders it against other stores).
__device__ inline void publish_q(uint64_t* qflag, int b, int32_t q) {
    if (qflag != nullptr && threadIdx.x == 0)
        __hip_atomic_store(&qflag[b], (uint64_t(1) << 32) | uint32_t(q), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

struct SelectArgs {
    int nb;
    int64_t chunks;
    int32_t alpha_ppm;
    const int32_t* sorted;
    const uint32_t* run_cnt;
    const uint32_t* run_start;
    const uint32_t* max_part;
    int32_t* q_out;
    int32_t* count_out;
    uint64_t* qflag;   // NULL when no apply workgroup waits
};

// Workgroup b of a selection: bucket b's size n_b and rank k_b (Eq. (3))
// from the run sizes, then the k_b-th smallest score of its runs, most
// significant 8-bit digit first from the top digit of the largest score.  A
// bucket of at most kSelNT * kKeep scores is gathered once (runs into LDS,
// then into registers) and kept across passes; a larger one is read from its
// runs on every pass.
__device__ int32_t select_bucket(const SelectArgs& A, int b) {
    const int nb = A.nb;
    const int64_t chunks = A.chunks;
    const int32_t alpha_ppm = A.alpha_ppm;
    const int32_t* __restrict__ sorted = A.sorted;
    int32_t* q_out = A.q_out;
    int32_t* count_out = A.count_out;
    (void)nb;
    extern __shared__ __align__(16) uint32_t stage[];   // [kSelNT * kKeep] the bucket's scores
    __shared__ uint32_t roff[kSortMaxChunks];           // where each run starts among the bucket's scores
    __shared__ uint32_t rcnt[kSortMaxChunks];           // its size
    __shared__ uint32_t rsrc[kSortMaxChunks];           // its first score's index in `sorted`
    __shared__ uint32_t hist[2][256];                   // digit histograms of alternate passes
    __shared__ uint32_t red[kSelWaves];
    __shared__ uint32_t pick[2][2];                     // digit and remaining rank of alternate passes
    const int t = threadIdx.x;
    const int lane = t % kWave, w = t / kWave;
    if (t < 256) hist[0][t] = 0;   // published by the barriers of the scans below
    uint32_t c = 0, m = 0, src = 0;
    if (t < chunks) {
        c = A.run_cnt[int64_t(b) * chunks + t];
        src = uint32_t(t * kChunk) + A.run_start[int64_t(b) * chunks + t];
        m = A.max_part[t];
    }
    uint32_t nbk;
    const uint32_t off = block_excl_scan<kSelNT, false>(c, 0u, red, &nbk);
    if (t < chunks) {
        roff[t] = off;
        rcnt[t] = c;
        rsrc[t] = src;
    }
    const uint32_t mx = block_reduce_max<kSelNT>(m, red);   // its barriers publish the run tables
    const int64_t k64 = (int64_t(1000000 - alpha_ppm) * (int64_t(nbk) + 1) + 999999) / 1000000;   // Eq. (3)
    if (t == 0) count_out[b] = int32_t(nbk);
    if (k64 > int64_t(nbk)) {
        if (t == 0) q_out[b] = MAPS_Q_INF;
        publish_q(A.qflag, b, MAPS_Q_INF);
        return MAPS_Q_INF;
    }
    int32_t k = int32_t(k64);
    const int top = mx >> 24 ? 24 : (mx >> 16 ? 16 : (mx >> 8 ? 8 : 0));
    const bool in_regs = nbk <= uint32_t(kSelNT) * kKeep;
    // Slot j = 4g + e of thread t holds score g * 4 * kSelNT + 4t + e of the
    // bucket (16-byte LDS reads); groups past n_b are skipped whole.
    uint32_t x[kKeep] = {};
    auto slot = [&](int j) { return uint32_t(j / 4) * (4 * kSelNT) + 4 * uint32_t(t) + uint32_t(j % 4); };
    uint32_t zeros = 0;   // the first pass's digit-0 count of this wavefront
    if (in_regs) {
        // wavefront w gathers runs w, w + kSelWaves, ...: the first 128
        // scores of kGatherRuns runs in flight per lane, longer runs' rest
        // after.  Lane q reads run q's table entry; the wavefront shares it.
        // Every score also enters the first pass's histogram (its top digit:
        // every score lies below 256 << top) as it arrives, so that pass
        // needs no loop of its own.
        for (int64_t r0 = w; r0 < chunks; r0 += int64_t(kSelWaves) * kGatherRuns) {
            const int64_t rq = r0 + int64_t(lane) * kSelWaves;
            const bool has = lane < kGatherRuns && rq < chunks;
            const uint32_t tc = has ? rcnt[rq] : 0u, ts = has ? rsrc[rq] : 0u, to = has ? roff[rq] : 0u;
            uint32_t v0[kGatherRuns], v1[kGatherRuns];
#pragma unroll
            for (int q = 0; q < kGatherRuns; ++q) {
                const uint32_t cn = __builtin_amdgcn_readlane(tc, q), s0 = __builtin_amdgcn_readlane(ts, q);
                v0[q] = uint32_t(lane) < cn ? uint32_t(sorted[s0 + lane]) : 0u;
                v1[q] = uint32_t(lane) + kWave < cn ? uint32_t(sorted[s0 + kWave + lane]) : 0u;
            }
#pragma unroll
            for (int q = 0; q < kGatherRuns; ++q) {
                const uint32_t cn = __builtin_amdgcn_readlane(tc, q), s0 = __builtin_amdgcn_readlane(ts, q);
                const uint32_t d0 = __builtin_amdgcn_readlane(to, q);
                if (uint32_t(lane) < cn) stage[d0 + lane] = v0[q];
                if (uint32_t(lane) + kWave < cn) stage[d0 + kWave + lane] = v1[q];
                hist_add(hist[0], uint32_t(lane) < cn, v0[q] >> top, zeros);
                hist_add(hist[0], uint32_t(lane) + kWave < cn, v1[q] >> top, zeros);
                for (uint32_t i0 = 2 * kWave; i0 < cn; i0 += kWave) {   // bounds uniform across the wavefront
                    const uint32_t i = i0 + lane;
                    const uint32_t v = i < cn ? uint32_t(sorted[s0 + i]) : 0u;
                    if (i < cn) stage[d0 + i] = v;
                    hist_add(hist[0], i < cn, v >> top, zeros);
                }
            }
        }
        hist_flush_zeros(hist[0], zeros);
        __syncthreads();
#pragma unroll
        for (int g = 0; g < kKeep / 4; ++g) {
            if (uint32_t(g) * (4 * kSelNT) >= nbk) break;
            const uint4 v = reinterpret_cast<const uint4*>(stage)[g * kSelNT + t];
            x[4 * g] = v.x;
            x[4 * g + 1] = v.y;
            x[4 * g + 2] = v.z;
            x[4 * g + 3] = v.w;
        }
    }
    // Pass p builds hist[p & 1] and picks into pick[p & 1]; the other
    // histogram is cleared meanwhile for the next pass.  Two barriers a pass:
    // after the histogram (before the pick) and after the pick (before
    // everyone reads it); a buffer is reused two passes later, past both.
    uint32_t prefix = 0;
    int pass = 0;
    for (int shift = top; shift >= 0; shift -= 8, ++pass) {
        const int cur = pass & 1;
        if (t < 256) hist[cur ^ 1][t] = 0;   // last read by the pick of the previous pass
        if (!(in_regs && pass == 0)) {       // the gather built the first in-register pass
            zeros = 0;
            if (in_regs) {
#pragma unroll
                for (int j = 0; j < kKeep; ++j) {
                    if (j % 4 == 0 && uint32_t(j / 4) * (4 * kSelNT) >= nbk) break;
                    const uint32_t y = x[j] >> shift;
                    hist_add(hist[cur], slot(j) < nbk && (y >> 8) == prefix, y & 255u, zeros);
                }
            } else {
                for (int64_t r = w; r < chunks; r += kSelWaves) {
                    const uint32_t cn = rcnt[r], s0 = rsrc[r];
                    for (uint32_t i0 = 0; i0 < cn; i0 += kWave) {   // bounds uniform across the wavefront
                        const uint32_t i = i0 + lane;
                        const uint32_t y = i < cn ? uint32_t(sorted[s0 + i]) >> shift : 0u;
                        hist_add(hist[cur], i < cn && (y >> 8) == prefix, y & 255u, zeros);
                    }
                }
            }
            hist_flush_zeros(hist[cur], zeros);
            __syncthreads();
        }
        if (t < kWave) pick_digit(hist[cur], k, pick[cur]);
        __syncthreads();
        prefix = (prefix << 8) | pick[cur][0];
        k = int32_t(pick[cur][1]);
    }
    if (t == 0) q_out[b] = int32_t(prefix);
    publish_q(A.qflag, b, int32_t(prefix));
    return int32_t(prefix);
}

// The selection alone: one workgroup per bucket.
__global__ __launch_bounds__(kSelNT) void cal_bucket_select(SelectArgs A) { (void)select_bucket(A, int(blockIdx.x)); }

struct ApplyArgs {
    const int32_t* edges;
    const int32_t* pred;
    int64_t m;
    int32_t u_max;
    int32_t* U;
    uint32_t* dev_err;
    uint32_t max_spins;   // polls of a quantile before the apply workgroup selects it itself
};

constexpr int kApplyFusedPer = 8;              // bounds per thread of a fused apply workgroup
constexpr uint32_t kMaxSpins = 1u << 14;       // polls of a quantile before selecting it locally (about 1 ms)
static_assert(2 * kSelStageBytes > 160 * 1024, "one workgroup of the fused launch per CU");
static_assert(kFastBuckets <= kSelNT, "one waiting thread per bucket");

// Apply workgroup j of ga in the fused launch (Eq. (4)): its first
// predictions are loaded and their buckets found while the selection runs;
// then thread i < nb waits (bounded) for bucket i's published quantile, and
// the workgroup writes its bounds, then the rest of its share.  A quantile
// still missing after the bounded wait (its selecting workgroup not yet
// resident: the device is shared, or did not hold the whole launch) is
// selected by this workgroup itself from the same sorted runs -- the same
// deterministic computation, so the same value -- so the launch completes
// and is exact whether or not its workgroups run at the same time.
__device__ void apply_after_select(const SelectArgs& S, const ApplyArgs& A, int j, int ga) {
    extern __shared__ __align__(16) uint32_t stage[];
    __shared__ uint32_t missing[kFastBuckets / 32];   // buckets whose quantile did not arrive
    const int nb = S.nb, ne = nb - 1;
    const int t = threadIdx.x;
    int32_t* le = reinterpret_cast<int32_t*>(stage);   // [ne] edges
    int32_t* lq = le + ne;                             // [nb] quantiles
    constexpr int kA = kApplyFusedPer;
    const int64_t stride = int64_t(ga) * kSelNT * kA;
    int32_t p[kA];
    int bk[kA];
    auto fetch = [&](int64_t c0) {
#pragma unroll
        for (int i = 0; i < kA; ++i) {
            const int64_t x = c0 + int64_t(i) * kSelNT + t;
            p[i] = x < A.m ? A.pred[x] : -1;
        }
    };
    auto emit = [&](int64_t c0) {
#pragma unroll
        for (int i = 0; i < kA; ++i) {
            const int64_t x = c0 + int64_t(i) * kSelNT + t;
            if (x >= A.m) continue;
            int32_t out = -1;   // no prediction: no bound
            if (p[i] >= 0) {
                const int32_t qb = lq[bk[i]];
                const int64_t v = int64_t(p[i]) + qb;   // Eq. (4)
                out = (qb == MAPS_Q_INF || v > A.u_max) ? A.u_max : int32_t(v);
            }
            A.U[x] = out;
        }
    };
    int64_t c0 = int64_t(j) * kSelNT * kA;
    fetch(c0);
    for (int i = t; i < ne; i += kSelNT) le[i] = A.edges[i];
    __syncthreads();
    buckets_of<kA>(le, ne, p, bk);
    if (t < kFastBuckets / 32) missing[t] = 0;
    __syncthreads();
    // nb <= kFastBuckets = kSelNT: thread i waits for bucket i
    uint64_t v = uint64_t(1) << 32;
    if ((t & ~(kWave - 1)) < nb) {   // wavefronts past nb: nothing to wait for
        uint32_t spins = 0;
        for (;;) {   // device-coherent polls, no cache invalidation
            v = t < nb ? __hip_atomic_load(&S.qflag[t], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                       : (uint64_t(1) << 32);
            if (__all(int(v >> 32) != 0)) break;
            if (++spins > A.max_spins) break;
            __builtin_amdgcn_s_sleep(8);
        }
        if (t < nb && (v >> 32) == 0) atomicOr(&missing[t / 32], 1u << (t % 32));
    }
    __syncthreads();
    int32_t q_own = int32_t(uint32_t(v));   // thread i < nb: bucket i's quantile
    bool any = false;
    for (int w = 0; w < kFastBuckets / 32; ++w) any |= missing[w] != 0;
    if (any) {   // uniform: every thread read the same bitmap
        for (int b = 0; b < nb; ++b) {
            if (!((missing[b / 32] >> (b % 32)) & 1u)) continue;
            const int32_t qb = select_bucket(S, b);   // overwrites `stage`: edges reloaded below
            if (t == b) q_own = qb;
        }
        __syncthreads();
        for (int i = t; i < ne; i += kSelNT) le[i] = A.edges[i];
    }
    if (t < nb) lq[t] = q_own;
    __syncthreads();
    emit(c0);
    for (c0 += stride; c0 < A.m; c0 += stride) {
        fetch(c0);
        buckets_of<kA>(le, ne, p, bk);
        emit(c0);
    }
}

// Selection and bounds in one launch: workgroups [0, nb) select, the rest
// apply.  Every workgroup holds more than half of a CU's LDS and the grid is
// at most the CU count, so normally all of them are resident at once and the
// apply workgroups find every quantile published; when not, they select the
// missing ones themselves after a bounded wait (no workgroup waits without
// bound on another).
__global__ __launch_bounds__(kSelNT) void cal_select_apply(SelectArgs S, ApplyArgs A) {
    if (int(blockIdx.x) < S.nb) select_bucket(S, int(blockIdx.x));
    else apply_after_select(S, A, int(blockIdx.x) - S.nb, int(gridDim.x) - S.nb);
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
// kSortMaxChunks chunks of kChunk residuals): chunks sorted by bucket, then
// one workgroup per bucket.
// When the grid fits the CUs, the bounds are written by extra workgroups of
// the selection's launch (*applied = true).
maps_status calibrate_fast(const int32_t* pred, const int32_t* truth, int64_t n, const int32_t* edges, int32_t nb,
                           int32_t alpha_ppm, int32_t* q_out, int32_t* count_out, const ApplyArgs& apply,
                           uint32_t* dev_err, void* workspace, hipStream_t stream, bool* applied) {
    const FastWorkspace w = fast_carve(workspace, n, nb);
    const int64_t chunks = sort_chunks(n);
    *applied = false;
    if (n > 0) {
        const size_t lds_sort = size_t(kChunk) * 4 + size_t(3 * nb - 1) * 4;   // chunk, edges, run sizes and starts
        allow_dynamic_lds(cal_chunk_sort, lds_sort);
        hipLaunchKernelGGL(cal_chunk_sort, dim3(unsigned(chunks)), dim3(kSortNT), lds_sort, stream, pred, truth, n,
                           edges, nb, chunks, w.run_cnt, w.run_start, w.max_part, w.sorted, w.qflag, dev_err);
        MAPS_CHECK_LAUNCH();
    }
    SelectArgs S{nb, chunks, alpha_ppm, w.sorted, w.run_cnt, w.run_start, w.max_part, q_out, count_out, nullptr};
    const int cus = device_compute_units();
    const int64_t per_wg = int64_t(kSelNT) * kApplyFusedPer;
    // the flags are cleared by the chunk sort, so the fused launch needs n > 0
    if (n > 0 && apply.m > 0 && int64_t(nb) + 1 <= cus) {
        const int64_t need = (apply.m + per_wg - 1) / per_wg;
        const int64_t ga = need < cus - nb ? need : cus - nb;
        S.qflag = w.qflag;
        allow_dynamic_lds(cal_select_apply, kSelStageBytes);
        hipLaunchKernelGGL(cal_select_apply, dim3(unsigned(nb + ga)), dim3(kSelNT), kSelStageBytes, stream, S,
                           apply);
        MAPS_CHECK_LAUNCH();
        *applied = true;
        return MAPS_OK;
    }
    allow_dynamic_lds(cal_bucket_select, kSelStageBytes);
    hipLaunchKernelGGL(cal_bucket_select, dim3(unsigned(nb)), dim3(kSelNT), kSelStageBytes, stream, S);
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
    bool applied = false;
    if (fast_path(n, nb)) {
        // MAPS_CAL_SPIN_LIMIT (tests only) lowers the bounded wait, so that the
        // local selection of missing quantiles is exercised
        const char* spin_env = getenv("MAPS_CAL_SPIN_LIMIT");
        const uint32_t spins = spin_env ? uint32_t(strtoul(spin_env, nullptr, 10)) : kMaxSpins;
        const ApplyArgs apply{edges, apply_pred, m, u_max, U_out, dev_err, spins};
        const maps_status st = calibrate_fast(pred, truth, n, edges, nb, alpha_ppm, q_out, count_out, apply, dev_err,
                                              workspace, stream, &applied);
        if (st != MAPS_OK) return st;
    } else {
        const maps_status st =
            calibrate_general(pred, truth, n, edges, nb, alpha_ppm, q_out, count_out, dev_err, workspace, stream);
        if (st != MAPS_OK) return st;
    }
    if (m > 0 && !applied) {
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



// ---------------------------------------------------------------------------
// Calibration without a caller workspace: the scratch lives in a file-scope
// device array (one per GPU, held until the process ends).  Host code never
// passes the array's name to a kernel: its device address is looked up once
// per device with hipGetSymbolAddress.
// ---------------------------------------------------------------------------
namespace {

constexpr size_t kScratchBytes = MAPS_CALIBRATE_NOALLOC_BYTES;
static __device__ __align__(256) char scratch[kScratchBytes];

// Device address of `scratch` on the current device (nullptr on failure).
void* scratch_address() {
    static std::mutex mu;
    static std::unordered_map<int, void*> addr;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return nullptr;
    std::lock_guard<std::mutex> lock(mu);
    auto it = addr.find(dev);
    if (it != addr.end()) return it->second;
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess) {
        (void)hipGetLastError();
        return nullptr;
    }
    addr[dev] = p;
    return p;
}

}  // namespace

extern "C" maps_status maps_calibrate_noalloc(const int32_t* pred, const int32_t* truth, int64_t n,
                                              const int32_t* edges, int32_t nb, int32_t alpha_ppm,
                                              int32_t* q_out, int32_t* count_out, const int32_t* apply_pred,
                                              int64_t m, int32_t u_max, int32_t* U_out, uint32_t* dev_err,
                                              hipStream_t stream) {
    if (n < 0 || m < 0 || nb < 1 || nb > 65536 || u_max < 0) return MAPS_E_SIZE;
    if (maps_calibrate_workspace_size(n, nb) > kScratchBytes) return MAPS_E_SIZE;
    void* ws = scratch_address();
    if (!ws) return MAPS_E_HIP;
    return maps_calibrate(pred, truth, n, edges, nb, alpha_ppm, q_out, count_out, apply_pred, m, u_max, U_out,
                          dev_err, ws, kScratchBytes, stream);
}
