// Incremental sliding-window calibration (Sec. 3.2: the calibration set is
// the most recent completed requests; Sec. 4: a window of 500) on gfx950.
//
// A persistent state holds, per length bucket, the number of completions it
// has seen and a ring of its last `window` nonconformity scores.  Appending a
// batch of completions touches only the ring slots of the newest entries of
// each bucket; the bounds of a batch of requests then come from each bucket's
// current window.  Nothing regroups the whole log.
//
//   win_hist     one workgroup per chunk of 1,024 new completions: bucket of
//                each (edges in LDS, binary search), kept as a 16-bit id, and
//                the chunk's count per bucket (LDS atomics on nb counters).
//   win_place    one workgroup per bucket: the bucket's new entries before
//                each chunk (a scan over the chunks, kept in LDS for appends
//                of up to 1,024 chunks), then only the chunks
//                that hold its last `window` new entries are visited, 16 at a
//                time: the entries of the bucket are ranked in log order
//                (ballots and a prefix over the wavefronts) and written to
//                their ring slots (count + rank) mod window; finally the
//                count grows.  Entries that a later entry of the same append
//                would overwrite are not written, so no slot is written twice.
//   win_select   one workgroup per bucket: the k-th smallest of its min(count,
//                window) scores, k = ceil((1 - alpha)(n_w + 1)) (Eq. (3)), by an
//                MSB-first radix select over LDS histograms, from the highest
//                byte the largest score uses, each pass's digit found by one
//                wavefront's scan of the 256 bins; infinite when k > n_w.
//   win_bounds   grid-stride: the bound of Eq. (4) for every request from the
//                quantile of its prediction's bucket.
#include "maps_internal.hpp"

namespace maps {
namespace {

constexpr uint32_t kWinMagic = 0x57494E53u;   // "WINS"
constexpr int kChunk = 1024;
constexpr int kHistNT = 1024;
constexpr int kPlaceNT = 1024;
constexpr int kSelNT = 1024;
constexpr int kBoundNT = 256;

struct WinHeader {
    uint32_t magic;
    int32_t nb, window, pad;
};

struct WinLayout {
    size_t off_count, off_ring, bytes;
};

__host__ __device__ inline WinLayout win_layout(int32_t nb, int32_t window) {
    WinLayout l;
    l.off_count = 256;
    l.off_ring = l.off_count + align256(size_t(nb) * sizeof(int64_t));
    l.bytes = l.off_ring + align256(size_t(nb) * size_t(window) * sizeof(int32_t));
    return l;
}

__device__ inline int32_t bucket_of(int32_t pred, const int32_t* edges, int32_t nb) {
    // #{edges <= pred}: the first edge above pred
    int32_t lo = 0, hi = nb - 1;
    while (lo < hi) {
        const int32_t mid = (lo + hi) >> 1;
        if (edges[mid] <= pred) lo = mid + 1;
        else hi = mid;
    }
    return lo;
}

__device__ inline bool state_ok(const char* state, int32_t nb, int32_t window) {
    const WinHeader* h = reinterpret_cast<const WinHeader*>(state);
    return h->magic == kWinMagic && h->nb == nb && h->window == window;
}

__global__ void win_reset(char* state, int32_t nb, int32_t window) {
    const WinLayout l = win_layout(nb, window);
    int64_t* count = reinterpret_cast<int64_t*>(state + l.off_count);
    for (int32_t b = blockIdx.x * blockDim.x + threadIdx.x; b < nb; b += gridDim.x * blockDim.x) count[b] = 0;
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        WinHeader* h = reinterpret_cast<WinHeader*>(state);
        h->magic = kWinMagic;
        h->nb = nb;
        h->window = window;
        h->pad = 0;
    }
}

struct AppendArgs {
    char* state;
    int32_t nb, window;
    const int32_t* pred;
    const int32_t* truth;
    int64_t k;
    const int32_t* edges;
    uint16_t* bid;      // workspace [k]
    int32_t* ccount;    // workspace [chunks][nb]
    int32_t chunks;
    uint32_t* dev_err;
};

__global__ __launch_bounds__(kHistNT) void win_hist(AppendArgs a) {
    extern __shared__ int32_t sh[];
    int32_t* edges = sh;               // nb - 1
    int32_t* cnt = sh + a.nb;          // nb
    const int32_t nb = a.nb;
    bool unsorted = false, neg = false;
    for (int32_t j = threadIdx.x; j < nb; j += kHistNT) {
        cnt[j] = 0;
        if (j < nb - 1) {
            edges[j] = a.edges[j];
            if (j > 0 && a.edges[j] < a.edges[j - 1]) unsorted = true;
        }
    }
    __syncthreads();
    const int64_t i = int64_t(blockIdx.x) * kChunk + threadIdx.x;
    if (i < a.k) {
        const int32_t p = a.pred[i], t = a.truth[i];
        neg = p < 0 || t < 0;
        const int32_t b = bucket_of(p, edges, nb);
        a.bid[i] = uint16_t(b);
        atomicAdd(&cnt[b], 1);
    }
    if (unsorted && blockIdx.x == 0) raise_error(a.dev_err, MAPS_ERR_EDGES_UNSORTED);
    if (__builtin_amdgcn_ballot_w64(neg) != 0 && threadIdx.x % kWave == 0) raise_error(a.dev_err, MAPS_ERR_NEG_LEN);
    __syncthreads();
    for (int32_t j = threadIdx.x; j < nb; j += kHistNT) a.ccount[int64_t(blockIdx.x) * nb + j] = cnt[j];
}

// Bucket b's workgroup.  The bucket's entries before each chunk come from a
// scan over the chunks of its column of ccount: held in LDS when the append
// has at most kPlaceNT chunks (kLds), else written over the column itself
// (the column is the workgroup's alone).  Only the chunks that hold one of
// the bucket's last `window` new entries are visited, kPlaceGroup of them at
// a time: thread t takes entry t of each, the wavefronts' ballots rank the
// entries inside each chunk, and a prefix over the wavefronts (one row of 16
// lanes per chunk) places them.  Every load of a group is issued before the
// group's first wait.
constexpr int kPlaceGroup = 16;   // chunks ranked together
constexpr int kPlaceWaves = kPlaceNT / kWave;
static_assert(kPlaceWaves == 16, "one DPP row of 16 lanes holds a chunk's wavefront counts");
static_assert(kPlaceGroup * kPlaceWaves <= kPlaceNT, "one thread per (chunk, wavefront) of a group");

template <bool kLds>
__global__ __launch_bounds__(kPlaceNT) void win_place(AppendArgs a) {
    __shared__ int32_t tmp[kPlaceWaves];
    __shared__ int32_t wcnt[kPlaceGroup * kPlaceWaves];   // bucket entries per (chunk of the group, wavefront)
    __shared__ int32_t spre[kLds ? kPlaceNT : 1];         // kLds: the bucket's entries before chunk c
    __shared__ int32_t first_active;
    const int32_t b = blockIdx.x, nb = a.nb, W = a.window;
    const int tid = threadIdx.x, lane = tid % kWave, wid = tid / kWave;
    const WinLayout l = win_layout(nb, W);
    int64_t* count = reinterpret_cast<int64_t*>(a.state + l.off_count);
    int32_t* ring = reinterpret_cast<int32_t*>(a.state + l.off_ring) + int64_t(b) * W;
    int32_t* pre = a.ccount + b;   // chunk c at pre[c * nb]
    // the header, the bucket's count and (kLds) this thread's chunk count are loaded together
    const int64_t c0 = count[b];
    const int32_t mine = kLds && tid < a.chunks ? pre[int64_t(tid) * nb] : 0;
    if (!state_ok(a.state, nb, W)) {   // not reset for these (nb, window)
        if (b == 0 && tid == 0) raise_error(a.dev_err, MAPS_ERR_SNAPSHOT);
        return;
    }
    int32_t total;
    if constexpr (kLds) {
        const int32_t run = block_excl_scan<kPlaceNT, false>(mine, 0, tmp, &total);
        spre[tid] = run;
    } else {
        total = block_scan<kPlaceNT, false, false, true, int32_t>(
            a.chunks, 0, [&](int64_t c) { return pre[c * nb]; }, [&](int64_t c, int32_t v) { pre[c * nb] = v; },
            tmp);
    }
    auto start_of = [&](int32_t c) { return kLds ? spre[c] : pre[int64_t(c) * nb]; };
    const int32_t keep = total - W;   // entries ranked below keep are overwritten within this append
    // ring slot of rank r: (c0 + r) mod W, with c0 reduced once; base + r < W + 2^31 fits 32 unsigned bits
    const uint32_t base = uint32_t(c0 % W);
    // the first chunk holding an entry of rank >= keep: the first c whose next chunk starts above keep
    if (tid == 0) first_active = a.chunks;
    __syncthreads();
    for (int32_t c = tid; c < a.chunks; c += kPlaceNT) {
        const int32_t next = c + 1 < a.chunks ? start_of(c + 1) : total;
        if (next > keep && next > start_of(c)) atomicMin(&first_active, c);
    }
    __syncthreads();
    for (int32_t g0 = first_active; g0 < a.chunks; g0 += kPlaceGroup) {
        bool hit[kPlaceGroup];
        int32_t before_lane[kPlaceGroup], t[kPlaceGroup], p[kPlaceGroup], start[kPlaceGroup];
#pragma unroll
        for (int j = 0; j < kPlaceGroup; ++j) {
            const int64_t i = int64_t(g0 + j) * kChunk + tid;
            hit[j] = g0 + j < a.chunks && i < a.k && a.bid[i] == b;
        }
#pragma unroll
        for (int j = 0; j < kPlaceGroup; ++j) {
            const int64_t i = int64_t(g0 + j) * kChunk + tid;
            t[j] = hit[j] ? a.truth[i] : 0;
            p[j] = hit[j] ? a.pred[i] : 0;
            start[j] = g0 + j < a.chunks ? start_of(g0 + j) : 0;
            const uint64_t bal = __builtin_amdgcn_ballot_w64(hit[j]);
            before_lane[j] = __popcll(bal & ((uint64_t(1) << lane) - 1));
            if (lane == 0) wcnt[j * kPlaceWaves + wid] = __popcll(bal);
        }
        __syncthreads();
        // exclusive prefix over the wavefronts of each chunk: thread (j, w) scans row j's 16 counts
        if (tid < kPlaceGroup * kPlaceWaves) {
            const int32_t v = wcnt[tid];
            int32_t incl = v;
            incl += dpp_move<kDppRowShr1, 0xf>(0, incl);
            incl += dpp_move<kDppRowShr2, 0xf>(0, incl);
            incl += dpp_move<kDppRowShr4, 0xf>(0, incl);
            incl += dpp_move<kDppRowShr8, 0xf>(0, incl);
            wcnt[tid] = incl - v;   // each thread rewrites only its own entry
        }
        __syncthreads();
#pragma unroll
        for (int j = 0; j < kPlaceGroup; ++j) {
            // rank among all new entries of the bucket (0-based, log order)
            const int32_t r = start[j] + wcnt[j * kPlaceWaves + wid] + before_lane[j];
            if (hit[j] && r >= keep) ring[(base + uint32_t(r)) % uint32_t(W)] = t[j] > p[j] ? t[j] - p[j] : 0;
        }
        __syncthreads();   // wcnt is reused by the next group
    }
    if (tid == 0) count[b] = c0 + total;
}

__device__ inline int64_t conformal_rank(int64_t n, int32_t alpha_ppm) {
    return ((int64_t(1000000) - alpha_ppm) * (n + 1) + 999999) / 1000000;
}

// The digit of the next radix pass, found by wavefront 0: lane l holds bins
// 4l .. 4l + 3, a wavefront scan gives the count below each lane, and the one
// lane whose range holds `rank` walks its four bins.  sel = {digit, rank
// within the digit}.
__device__ inline void pick_digit(const int32_t* hist, int32_t rank, int32_t* sel) {
    const int lane = threadIdx.x % kWave;
    const int32_t h0 = hist[4 * lane], h1 = hist[4 * lane + 1], h2 = hist[4 * lane + 2], h3 = hist[4 * lane + 3];
    const int32_t sum = h0 + h1 + h2 + h3;
    const int32_t incl = wave_incl_scan_add(sum);
    int32_t acc = incl - sum;
    if (acc < rank && rank <= incl) {
        int32_t d = 4 * lane;
        if (acc + h0 < rank) {
            acc += h0;
            ++d;
            if (acc + h1 < rank) {
                acc += h1;
                ++d;
                if (acc + h2 < rank) {
                    acc += h2;
                    ++d;
                }
            }
        }
        sel[0] = d;
        sel[1] = rank - acc;
    }
}

__global__ __launch_bounds__(kSelNT) void win_select(const char* state, int32_t nb, int32_t W, int32_t alpha_ppm,
                                                     int32_t* q, uint32_t* dev_err) {
    extern __shared__ int32_t vals[];   // W
    __shared__ int32_t hist[256];
    __shared__ int32_t sel[2];          // digit, remaining rank
    __shared__ uint32_t vmax;
    const int32_t b = blockIdx.x;
    if (!state_ok(state, nb, W)) {
        if (threadIdx.x == 0) {
            q[b] = MAPS_Q_INF;
            if (b == 0) raise_error(dev_err, MAPS_ERR_SNAPSHOT);
        }
        return;
    }
    const WinLayout l = win_layout(nb, W);
    const int64_t c = reinterpret_cast<const int64_t*>(state + l.off_count)[b];
    const int32_t nw = int32_t(c < W ? c : W);
    const int64_t k = conformal_rank(nw, alpha_ppm);
    if (k > nw) {   // also the empty window
        if (threadIdx.x == 0) q[b] = MAPS_Q_INF;
        return;
    }
    const int32_t* ring = reinterpret_cast<const int32_t*>(state + l.off_ring) + int64_t(b) * W;
    if (threadIdx.x == 0) vmax = 0;
    __syncthreads();
    // the window is the ring's first nw slots (all W once the bucket has wrapped); scores are >= 0
    uint32_t m = 0;
    for (int32_t j = threadIdx.x; j < nw; j += kSelNT) {
        const int32_t v = ring[j];
        vals[j] = v;
        m = m > uint32_t(v) ? m : uint32_t(v);
    }
    m = wave_reduce_max(m);
    if (threadIdx.x % kWave == 0) atomicMax(&vmax, m);
    __syncthreads();
    // passes start at the highest byte the largest score uses: the bytes above it are 0 in every score
    const uint32_t top = vmax;
    const int first = top >> 24 ? 24 : top >> 16 ? 16 : top >> 8 ? 8 : 0;
    uint32_t prefix = 0, mask = first == 24 ? 0u : ~0u << (first + 8);
    int32_t rank = int32_t(k);   // 1-indexed among the values matching prefix under mask
    for (int shift = first; shift >= 0; shift -= 8) {
        for (int j = threadIdx.x; j < 256; j += kSelNT) hist[j] = 0;
        __syncthreads();
        for (int32_t j = threadIdx.x; j < nw; j += kSelNT) {
            const uint32_t v = uint32_t(vals[j]);
            if ((v & mask) == prefix) atomicAdd(&hist[(v >> shift) & 255], 1);
        }
        __syncthreads();
        if (threadIdx.x < kWave) pick_digit(hist, rank, sel);
        __syncthreads();
        prefix |= uint32_t(sel[0]) << shift;
        mask |= 255u << shift;
        rank = sel[1];
        __syncthreads();
    }
    if (threadIdx.x == 0) q[b] = int32_t(prefix);
}

__global__ __launch_bounds__(kBoundNT) void win_bounds(const int32_t* edges_g, int32_t nb, const int32_t* q_g,
                                                       const int32_t* pred, int64_t m, int32_t u_max, int32_t* U) {
    extern __shared__ int32_t sh[];
    int32_t* edges = sh;
    int32_t* q = sh + nb;
    for (int32_t j = threadIdx.x; j < nb; j += kBoundNT) {
        if (j < nb - 1) edges[j] = edges_g[j];
        q[j] = q_g[j];
    }
    __syncthreads();
    for (int64_t i = int64_t(blockIdx.x) * kBoundNT + threadIdx.x; i < m; i += int64_t(gridDim.x) * kBoundNT) {
        const int32_t p = pred[i];
        if (p < 0) {
            U[i] = -1;
            continue;
        }
        const int32_t qb = q[bucket_of(p, edges, nb)];
        if (qb == MAPS_Q_INF) U[i] = u_max;
        else {
            const int64_t u = int64_t(p) + qb;
            U[i] = int32_t(u < u_max ? u : u_max);
        }
    }
}

bool header_ok_host(int32_t nb, int32_t window) {
    return nb >= 1 && nb <= MAPS_MAX_WINDOW_BUCKETS && window >= 1 && window <= MAPS_MAX_WINDOW;
}

}  // namespace
}  // namespace maps

using namespace maps;

extern "C" size_t maps_window_state_bytes(int32_t nb, int32_t window) {
    if (!header_ok_host(nb, window)) return 0;
    return win_layout(nb, window).bytes;
}

extern "C" size_t maps_window_append_workspace_size(int64_t k, int32_t nb) {
    if (k < 0 || nb < 1 || nb > MAPS_MAX_WINDOW_BUCKETS) return 0;
    const int64_t chunks = (k + kChunk - 1) / kChunk;
    return align256(size_t(k) * sizeof(uint16_t)) + align256(size_t(chunks) * nb * sizeof(int32_t));
}

extern "C" maps_status maps_window_reset(void* state, size_t state_bytes, int32_t nb, int32_t window,
                                         hipStream_t stream) {
    if (!header_ok_host(nb, window)) return MAPS_E_SIZE;
    if (!state) return MAPS_E_NULL;
    if (state_bytes < win_layout(nb, window).bytes) return MAPS_E_BUFFER;
    hipLaunchKernelGGL(win_reset, dim3(unsigned((nb + 255) / 256)), dim3(256), 0, stream, static_cast<char*>(state),
                       nb, window);
    MAPS_CHECK_LAUNCH();
    return MAPS_OK;
}

extern "C" maps_status maps_window_append(void* state, size_t state_bytes, int32_t nb, int32_t window,
                                          const int32_t* pred, const int32_t* truth, int64_t k,
                                          const int32_t* edges, uint32_t* dev_err, void* workspace,
                                          size_t workspace_bytes, hipStream_t stream) {
    if (!header_ok_host(nb, window) || k < 0 || k > INT32_MAX) return MAPS_E_SIZE;
    if (!state || !dev_err || (k > 0 && (!pred || !truth || !workspace)) || (nb > 1 && !edges)) return MAPS_E_NULL;
    if (state_bytes < win_layout(nb, window).bytes) return MAPS_E_BUFFER;
    if (k == 0) return MAPS_OK;
    if (workspace_bytes < maps_window_append_workspace_size(k, nb)) return MAPS_E_WORKSPACE;
    const int64_t chunks = (k + kChunk - 1) / kChunk;
    char* w = static_cast<char*>(workspace);
    AppendArgs a{static_cast<char*>(state), nb, window, pred, truth, k, edges, reinterpret_cast<uint16_t*>(w),
                 reinterpret_cast<int32_t*>(w + align256(size_t(k) * sizeof(uint16_t))), int32_t(chunks), dev_err};
    const size_t lds = size_t(2) * nb * sizeof(int32_t);
    allow_dynamic_lds(win_hist, lds);
    hipLaunchKernelGGL(win_hist, dim3(unsigned(chunks)), dim3(kHistNT), lds, stream, a);
    MAPS_CHECK_LAUNCH();
    if (chunks <= kPlaceNT) hipLaunchKernelGGL(win_place<true>, dim3(unsigned(nb)), dim3(kPlaceNT), 0, stream, a);
    else hipLaunchKernelGGL(win_place<false>, dim3(unsigned(nb)), dim3(kPlaceNT), 0, stream, a);
    MAPS_CHECK_LAUNCH();
    return MAPS_OK;
}

extern "C" maps_status maps_window_bounds(const void* state, size_t state_bytes, int32_t nb, int32_t window,
                                          int32_t alpha_ppm, const int32_t* edges, const int32_t* apply_pred,
                                          int64_t m, int32_t u_max, int32_t* q_out, int32_t* U_out,
                                          uint32_t* dev_err, hipStream_t stream) {
    if (!header_ok_host(nb, window) || m < 0 || u_max < 0) return MAPS_E_SIZE;
    if (alpha_ppm <= 0 || alpha_ppm >= 1000000) return MAPS_E_ALPHA;
    if (!state || !q_out || !dev_err || (nb > 1 && !edges) || (m > 0 && (!apply_pred || !U_out)))
        return MAPS_E_NULL;
    if (state_bytes < win_layout(nb, window).bytes) return MAPS_E_BUFFER;
    const size_t lds_sel = size_t(window) * sizeof(int32_t);
    allow_dynamic_lds(win_select, lds_sel);
    hipLaunchKernelGGL(win_select, dim3(unsigned(nb)), dim3(kSelNT), lds_sel, stream,
                       static_cast<const char*>(state), nb, window, alpha_ppm, q_out, dev_err);
    MAPS_CHECK_LAUNCH();
    if (m > 0) {
        const int64_t blocks = (m + kBoundNT - 1) / kBoundNT;
        const size_t lds = size_t(2) * nb * sizeof(int32_t);
        allow_dynamic_lds(win_bounds, lds);
        hipLaunchKernelGGL(win_bounds, dim3(unsigned(blocks < 2048 ? blocks : 2048)), dim3(kBoundNT), lds, stream,
                           edges, nb, q_out, apply_pred, m, u_max, U_out);
        MAPS_CHECK_LAUNCH();
    }
    return MAPS_OK;
}
