// Sliding-window calibration (Sec. 3.2: the calibration set is made of the
// most recent completed requests; Sec. 4: the 500 most recent) on gfx950.
//
// Request j is calibrated on its own set: the `window` (W) most recent entries
// of its bucket among the first seen[j] entries of the completion log.  With
// x_0, x_1, ... the scores of bucket b in log order, a request that saw c of
// them uses x_{max(0,c-W)} .. x_{c-1}; every position c = 0..n_b of every
// bucket therefore has one quantile, and each request looks its own up.
//
//   win_chunk_sort  per chunk of 4,096 log entries: scores and buckets, the
//                   chunk grouped by bucket with log order inside each group
//                   (a stable counting sort: each wavefront ranks its 64
//                   entries a round among equal buckets through ballots and
//                   keeps running counts per bucket in LDS, then per bucket a
//                   prefix over the wavefronts and over the buckets), and
//                   every group's size and start; each entry's bucket in log
//                   order, and per bucket and 64-entry sub-block of the chunk
//                   the bucket's entries before the sub-block;
//   win_row_scan    per bucket: the prefix over chunks of its group sizes
//                   (where each chunk's group starts in the bucket sequence);
//   win_scatter     every score to its place in its bucket's sequence (the
//                   buckets one after another); workgroup 0 also writes the
//                   per-bucket bases of the quantile table and of the select
//                   grid;
//   win_select      per run of C consecutive positions of one bucket: a
//                   wavelet matrix of the scores x_{c0-W} .. x_{c0+C-2} in LDS
//                   (one stable partition by each score bit, most significant
//                   first, with popcount rank directories); then one thread per
//                   position takes the k-th smallest score of its window, one
//                   rank step per bit;
//   win_apply       per request: its bucket, its position c (the bucket's
//                   entries before its chunk, then before its sub-block, then
//                   a count of its bucket among the at most 63 entries it saw
//                   of the sub-block: one line of bucket ids, 64 bytes with at
//                   most 256 buckets, else 128), the
//                   quantile and the bound (Eq. (4)).
// Every step is integer arithmetic, so the result is deterministic.
#include "maps_internal.hpp"

namespace maps {
namespace {

constexpr int kChunk = 4096;                    // log entries per sort workgroup
constexpr int kSortNT = 1024;
constexpr int kSortPer = kChunk / kSortNT;
constexpr int kSegs = kSortNT / kWave;          // one segment of kSortPer * 64 entries per wavefront
constexpr int kBucketsMax = MAPS_MAX_WINDOW_BUCKETS;
constexpr int kSelNT = 512;
constexpr int kSelPer = 3;                      // positions per select thread
constexpr int kSelC = kSelNT * kSelPer;         // positions per select workgroup
constexpr int kLevels = 31;                     // score bits (scores are non-negative int32)
constexpr int kSub = 64;                        // log entries per sub-block of the position table
constexpr int kSubs = kChunk / kSub;
constexpr int kApplyNT = 256;
constexpr int kApplyPer = 2;                   // requests per apply thread

struct WinWorkspace {
    int32_t* run_s;     // [n] scores, each chunk grouped by bucket
    uint16_t* run_b;    // [n] buckets, same order
    uint16_t* lb;       // [nch * kChunk] bucket of each log entry, log order (the tail past n unused);
                        //   one byte each when there are at most 256 buckets
    uint16_t* t64;      // [nb][nch][kSubs] entries of the bucket in the chunk before each sub-block
    int32_t* cnt;       // [nb][nch] group sizes
    int32_t* rs;        // [nb][nch] group starts inside the chunk
    int32_t* off;       // [nb][nch + 1] bucket position of each group; off[b][nch] = n_b
    int32_t* sub;       // [n] scores of bucket 0, then bucket 1, ... (log order inside each)
    int64_t* bstart;    // [nb] first entry of bucket b in sub
    int64_t* pbase;     // [nb] first quantile of bucket b in qw: sum_{b' < b} (n_b' + 1)
    int32_t* wstart;    // [nb + 1] first select workgroup of bucket b
    int32_t* qw;        // [n + nb] quantile at every position of every bucket
    size_t bytes;
};

WinWorkspace win_carve(void* base, int64_t n, int32_t nb) {
    WinWorkspace w;
    const int64_t nch = (n + kChunk - 1) / kChunk;
    size_t off = 0;
    char* p = static_cast<char*>(base);
    auto take = [&](size_t bytes) { char* r = p ? p + off : nullptr; off += align256(bytes); return r; };
    w.run_s = reinterpret_cast<int32_t*>(take(size_t(n) * 4));
    w.run_b = reinterpret_cast<uint16_t*>(take(size_t(n) * 2));
    w.lb = reinterpret_cast<uint16_t*>(take(size_t(nch) * kChunk * 2));
    w.t64 = reinterpret_cast<uint16_t*>(take(size_t(nb) * size_t(nch) * kSubs * 2));
    w.cnt = reinterpret_cast<int32_t*>(take(size_t(nb) * size_t(nch) * 4));
    w.rs = reinterpret_cast<int32_t*>(take(size_t(nb) * size_t(nch) * 4));
    w.off = reinterpret_cast<int32_t*>(take(size_t(nb) * size_t(nch + 1) * 4));
    w.sub = reinterpret_cast<int32_t*>(take(size_t(n) * 4));
    w.bstart = reinterpret_cast<int64_t*>(take(size_t(nb) * 8));
    w.pbase = reinterpret_cast<int64_t*>(take(size_t(nb) * 8));
    w.wstart = reinterpret_cast<int32_t*>(take(size_t(nb + 1) * 4));
    w.qw = reinterpret_cast<int32_t*>(take(size_t(n + nb) * 4));
    w.bytes = off;
    return w;
}

// Number of edges <= v among edges[0..ne-1].
__device__ inline int win_bucket(const int32_t* edges, int ne, int32_t v) {
    int lo = 0, hi = ne;
    while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (edges[mid] <= v) lo = mid + 1; else hi = mid;
    }
    return lo;
}

// Eq. (3): k = ceil((1 - alpha)(n + 1)) with alpha = alpha_ppm / 10^6.
__device__ inline int64_t win_rank(int64_t n, int32_t alpha_ppm) {
    return (int64_t(1000000 - alpha_ppm) * (n + 1) + 999999) / 1000000;
}

struct WinArgs {
    const int32_t* pred;
    const int32_t* truth;
    int64_t n;
    int64_t nch;
    const int32_t* edges;
    int32_t nb;
    int32_t window;
    int32_t alpha_ppm;
    WinWorkspace w;
    uint32_t* dev_err;
};

// ---------------------------------------------------------------------------
// 1. Each chunk grouped by bucket, log order inside each group
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kSortNT) void win_chunk_sort(WinArgs a) {
    __shared__ int32_t le[kBucketsMax - 1];
    __shared__ uint16_t seg[kSegs][kBucketsMax];   // entries of each bucket in each wave's segment
    __shared__ int32_t grp[kBucketsMax];           // chunk counts, then group starts
    __shared__ uint16_t locs[kChunk];              // chunk position of each grouped entry
    __shared__ int32_t tmp[kSortNT / kWave];
    const int ne = a.nb - 1;
    const int lane = threadIdx.x % kWave, wid = threadIdx.x / kWave;
    for (int i = threadIdx.x; i < ne; i += kSortNT) le[i] = a.edges[i];
    for (int i = threadIdx.x; i < kSegs * a.nb; i += kSortNT) seg[i / a.nb][i % a.nb] = 0;
    if (blockIdx.x == 0)
        for (int i = threadIdx.x; i + 1 < ne; i += kSortNT)
            if (a.edges[i] > a.edges[i + 1]) raise_error(a.dev_err, MAPS_ERR_EDGES_UNSORTED);
    __syncthreads();
    const int64_t base = int64_t(blockIdx.x) * kChunk;
    const int nbits = a.nb > 1 ? 32 - __clz(uint32_t(a.nb - 1)) : 0;
    const uint64_t below = (uint64_t(1) << lane) - 1u;
    int32_t s[kSortPer], b[kSortPer], rank[kSortPer];
    bool bad = false;
    // wave w owns the 256 entries [256 w, 256 w + 256) of the chunk, 64 a round
#pragma unroll
    for (int r = 0; r < kSortPer; ++r) {
        const int loc = wid * (kWave * kSortPer) + r * kWave + lane;
        const int64_t i = base + loc;
        const bool valid = i < a.n;
        s[r] = 0;
        b[r] = 0;
        if (valid) {
            const int32_t p = a.pred[i], t = a.truth[i];
            bad |= (p < 0) | (t < 0);
            const int64_t d = int64_t(t) - p;   // Eq. (2)
            s[r] = d <= 0 ? 0 : (d > INT32_MAX ? INT32_MAX : int32_t(d));
            b[r] = win_bucket(le, ne, p);
        }
        // lanes with the same bucket, bit by bit through ballots
        uint64_t peers = __ballot(valid);
        for (int bit = 0; bit < nbits; ++bit) {
            const bool one = (b[r] >> bit) & 1;
            const uint64_t m = __ballot(one);
            peers &= one ? m : ~m;
        }
        const int before = __popcll(peers & below);
        rank[r] = 0;
        if (valid) {
            // every lane of the group reads the running count before its
            // first lane adds the group (one wavefront: LDS operations in order)
            const int run = seg[wid][b[r]];
            rank[r] = run + before;
            if (before == 0) seg[wid][b[r]] = uint16_t(run + __popcll(peers));
        }
    }
    if (bad) raise_error(a.dev_err, MAPS_ERR_NEG_LEN);
    __syncthreads();
    // per bucket: the entries in earlier segments, and the chunk's count
    for (int bb = threadIdx.x; bb < a.nb; bb += kSortNT) {
        int acc = 0;
#pragma unroll
        for (int w = 0; w < kSegs; ++w) {
            const int v = seg[w][bb];
            seg[w][bb] = uint16_t(acc);
            acc += v;
        }
        grp[bb] = acc;
    }
    __syncthreads();
    // group starts (exclusive scan over buckets); sizes and starts to the tables
    const int64_t c = blockIdx.x;
    block_scan<kSortNT, false, false, true, int32_t>(
        a.nb, 0, [&](int64_t bb) { return grp[bb]; },
        [&](int64_t bb, int32_t v) {
            a.w.cnt[bb * a.nch + c] = grp[bb];
            a.w.rs[bb * a.nch + c] = v;
            grp[bb] = v;
        },
        tmp);
#pragma unroll
    for (int r = 0; r < kSortPer; ++r) {
        const int loc = wid * (kWave * kSortPer) + r * kWave + lane;
        const int64_t i = base + loc;
        if (i < a.n) {
            const int64_t pos = base + grp[b[r]] + seg[wid][b[r]] + rank[r];
            a.w.run_s[pos] = s[r];
            a.w.run_b[pos] = uint16_t(b[r]);
            if (a.nb <= 256) reinterpret_cast<uint8_t*>(a.w.lb)[i] = uint8_t(b[r]);
            else a.w.lb[i] = uint16_t(b[r]);
            locs[pos - base] = uint16_t(loc);
        }
    }
    __syncthreads();
    // per bucket and sub-block: the bucket's entries at chunk positions below
    // the sub-block (a search of the group's ascending positions)
    const int nvalid = a.n - base < kChunk ? int(a.n - base) : kChunk;
    for (int t = threadIdx.x; t < a.nb * kSubs; t += kSortNT) {
        const int bb = t / kSubs, sb = t % kSubs;
        const int g0 = grp[bb], g1 = bb + 1 < a.nb ? grp[bb + 1] : nvalid;
        const int bound = sb * kSub;
        int lo = g0, hi = g1;
        while (lo < hi) {
            const int mid = (lo + hi) >> 1;
            if (locs[mid] < bound) lo = mid + 1; else hi = mid;
        }
        a.w.t64[(int64_t(bb) * a.nch + c) * kSubs + sb] = uint16_t(lo - g0);
    }
}

// ---------------------------------------------------------------------------
// 2. Per bucket: where each chunk's group starts in the bucket's sequence
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void win_row_scan(WinArgs a) {
    __shared__ int32_t tmp[256 / kWave];
    const int64_t b = blockIdx.x;
    const int32_t* row = a.w.cnt + b * a.nch;
    int32_t* out = a.w.off + b * (a.nch + 1);
    const int32_t total = block_scan<256, false, false, true, int32_t>(
        a.nch, 0, [&](int64_t c) { return row[c]; }, [&](int64_t c, int32_t v) { out[c] = v; }, tmp);
    if (threadIdx.x == 0) out[a.nch] = total;
}

// ---------------------------------------------------------------------------
// 3. Scores to their bucket sequences; bases of the quantile table and grid
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kSortNT) void win_scatter(WinArgs a) {
    __shared__ int64_t bst[kBucketsMax];
    __shared__ int64_t tmp64[kSortNT / kWave];
    __shared__ int32_t tmp32[kSortNT / kWave];
    const int64_t stride = a.nch + 1;
    auto total = [&](int64_t b) { return int64_t(a.w.off[b * stride + a.nch]); };
    block_scan<kSortNT, false, false, true, int64_t>(
        a.nb, int64_t(0), total, [&](int64_t b, int64_t v) { bst[b] = v; }, tmp64);
    if (blockIdx.x == 0) {
        for (int b = threadIdx.x; b < a.nb; b += kSortNT) {
            a.w.bstart[b] = bst[b];
            a.w.pbase[b] = bst[b] + b;
        }
        const int32_t groups = block_scan<kSortNT, false, false, true, int32_t>(
            a.nb, 0, [&](int64_t b) { return int32_t((total(b) + kSelC) / kSelC); },   // ceil((n_b + 1) / C)
            [&](int64_t b, int32_t v) { a.w.wstart[b] = v; }, tmp32);
        if (threadIdx.x == 0) a.w.wstart[a.nb] = groups;
    }
    const int64_t c = blockIdx.x;
    if (c >= a.nch) return;
    const int64_t base = c * kChunk;
    const int64_t left = a.n - base;
    const int valid = left < kChunk ? int(left) : kChunk;
    for (int p = threadIdx.x; p < valid; p += kSortNT) {
        const int64_t b = a.w.run_b[base + p];
        const int64_t dst = bst[b] + a.w.off[b * stride + c] + (p - a.w.rs[b * a.nch + c]);
        a.w.sub[dst] = a.w.run_s[base + p];
    }
}

// ---------------------------------------------------------------------------
// 4. Quantile at every position: wavelet matrix over each run's windows
// ---------------------------------------------------------------------------
// Dynamic LDS of one select workgroup for windows of W: two score buffers of
// M = W + C - 1 entries, and per level the bit words and the ones before each
// word (M / 32 + 1 words, the last one empty).
struct SelLayout {
    int M, words;
    size_t off_bits, off_dir, off_zero, bytes;
};

__host__ __device__ inline SelLayout sel_layout(int32_t window) {
    SelLayout s;
    s.M = window + kSelC - 1;
    s.words = s.M / 32 + 1;
    s.off_bits = size_t(2) * s.M * 4;
    s.off_dir = s.off_bits + size_t(kLevels) * s.words * 4;
    s.off_zero = s.off_dir + size_t(kLevels) * s.words * 4;
    s.bytes = s.off_zero + kLevels * 4 + 64;
    return s;
}

__device__ inline int32_t rank1(const uint32_t* bits, const int32_t* dir, int i) {
    const int w = i >> 5;
    return dir[w] + __popc(bits[w] & ((1u << (i & 31)) - 1u));
}

__global__ __launch_bounds__(kSelNT) void win_select(WinArgs a) {
    extern __shared__ __align__(16) unsigned char sel_lds[];
    __shared__ int32_t tmp[kSelNT / kWave];
    __shared__ uint32_t tmpu[kSelNT / kWave];
    const SelLayout S = sel_layout(a.window);
    uint32_t* buf0 = reinterpret_cast<uint32_t*>(sel_lds);
    uint32_t* buf1 = buf0 + S.M;
    uint32_t* bits = reinterpret_cast<uint32_t*>(sel_lds + S.off_bits);
    int32_t* dir = reinterpret_cast<int32_t*>(sel_lds + S.off_dir);
    int32_t* zeros = reinterpret_cast<int32_t*>(sel_lds + S.off_zero);

    // the bucket of this workgroup: the last b with wstart[b] <= blockIdx
    const int32_t g = blockIdx.x;
    int32_t le_count = 0;
    for (int b = threadIdx.x; b < a.nb; b += kSelNT) le_count += a.w.wstart[b] <= g ? 1 : 0;
    const int32_t nle = block_reduce_add<kSelNT>(le_count, tmp);
    if (g >= a.w.wstart[a.nb]) return;   // past the last run (the grid is an upper bound)
    const int32_t b = nle - 1;
    const int64_t nb_b = a.w.off[int64_t(b) * (a.nch + 1) + a.nch];
    const int64_t j0 = int64_t(g - a.w.wstart[b]) * kSelC;
    const int64_t j1 = j0 + kSelC < nb_b + 1 ? j0 + kSelC : nb_b + 1;
    const int64_t W = a.window;
    const int64_t e0 = j0 - W > 0 ? j0 - W : 0;
    const int64_t e1 = j1 - 1 > e0 ? j1 - 1 : e0;
    const int M = int(e1 - e0);
    const int32_t* src = a.w.sub + a.w.bstart[b] + e0;
    uint32_t mx = 0;
    for (int i = threadIdx.x; i < M; i += kSelNT) {
        const uint32_t v = uint32_t(src[i]);
        buf0[i] = v;
        mx = mx > v ? mx : v;
    }
    mx = block_reduce_max<kSelNT>(mx, tmpu);
    const int L = mx ? 32 - __clz(mx) : 0;
    const int words = M / 32 + 1;

    // levels, most significant bit first: bit words, rank directory, stable partition
    uint32_t* cur = buf0;
    uint32_t* nxt = buf1;
    const int lane = threadIdx.x % kWave, wid = threadIdx.x / kWave;
    for (int l = 0; l < L; ++l) {
        const int bit = L - 1 - l;
        uint32_t* lb = bits + l * S.words;
        int32_t* ld = dir + l * S.words;
        for (int i0 = wid * kWave; i0 < words * 32; i0 += kSelNT) {
            const int i = i0 + lane;
            const bool one = i < M && ((cur[i] >> bit) & 1u);
            const uint64_t m = __ballot(one);
            if (lane == 0) lb[i0 >> 5] = uint32_t(m);
            if (lane == 32 && (i0 >> 5) + 1 < words) lb[(i0 >> 5) + 1] = uint32_t(m >> 32);
        }
        __syncthreads();
        if (wid == 0) {
            // ones before each word: a wavefront scan over the words, 64 at a time
            int32_t carry = 0;
            for (int w0 = 0; w0 < words; w0 += kWave) {
                const int w = w0 + lane;
                const int32_t c = w < words ? __popc(lb[w]) : 0;
                const int32_t incl = wave_incl_scan_add(c);
                if (w < words) ld[w] = carry + incl - c;
                carry += wave_last(incl);
            }
            if (lane == 0) zeros[l] = M - carry;
        }
        __syncthreads();
        const int32_t z = zeros[l];
        for (int i = threadIdx.x; i < M; i += kSelNT) {
            const uint32_t v = cur[i];
            const int32_t r1 = rank1(lb, ld, i);
            const int32_t dst = ((v >> bit) & 1u) ? z + r1 : i - r1;
            nxt[dst] = v;
        }
        __syncthreads();
        uint32_t* t = cur; cur = nxt; nxt = t;
    }

    // one position per thread: the k-th smallest score of entries [lo, hi)
    int32_t* out = a.w.qw + a.w.pbase[b];
#pragma unroll
    for (int r = 0; r < kSelPer; ++r) {
        const int64_t j = j0 + threadIdx.x + r * kSelNT;
        if (j >= j1) continue;
        int lo = int((j - W > 0 ? j - W : 0) - e0);
        int hi = int(j - e0);
        const int64_t nw = hi - lo;
        int64_t k = win_rank(nw, a.alpha_ppm);
        int32_t q = MAPS_Q_INF;
        if (k <= nw) {
            uint32_t v = 0;
            for (int l = 0; l < L; ++l) {
                const uint32_t* lb = bits + l * S.words;
                const int32_t* ld = dir + l * S.words;
                const int32_t r1lo = rank1(lb, ld, lo), r1hi = rank1(lb, ld, hi);
                const int32_t zin = (hi - lo) - (r1hi - r1lo);
                if (k <= zin) {
                    lo -= r1lo;
                    hi -= r1hi;
                } else {
                    k -= zin;
                    lo = zeros[l] + r1lo;
                    hi = zeros[l] + r1hi;
                    v |= 1u << (L - 1 - l);
                }
            }
            q = int32_t(v);
        }
        out[j] = q;
    }
}

// ---------------------------------------------------------------------------
// 5. Per request: its bucket position, quantile and bound
// ---------------------------------------------------------------------------
struct ApplyArgs {
    const int32_t* apply_pred;
    const int64_t* seen;
    int64_t m;
    int32_t u_max;
    int32_t* q_out;
    int32_t* U_out;
};

template <bool kByteIds>
__global__ __launch_bounds__(kApplyNT) void win_apply(WinArgs a, ApplyArgs r) {
    constexpr int kIdBytes = kByteIds ? 1 : 2;
    constexpr int kVecs = kSub * kIdBytes / 16;    // 16-byte loads per sub-block line
    constexpr int kPerWord = 4 / kIdBytes;
    __shared__ int32_t ledges[kBucketsMax - 1];
    __shared__ int64_t lpbase[kBucketsMax];
    const int ne = a.nb - 1;
    for (int i = threadIdx.x; i < ne; i += kApplyNT) ledges[i] = a.edges[i];
    for (int i = threadIdx.x; i < a.nb; i += kApplyNT) lpbase[i] = a.w.pbase[i];
    __syncthreads();
    bool bad = false;
    // kApplyPer requests per thread; the line of bucket ids depends only on
    // the seen count, so its loads go out before the bucket is known
    for (int64_t j0 = int64_t(blockIdx.x) * (kApplyNT * kApplyPer); j0 < r.m;
         j0 += int64_t(gridDim.x) * (kApplyNT * kApplyPer)) {
        int32_t p[kApplyPer], b[kApplyPer], rem[kApplyPer];
        int64_t seen[kApplyPer], ch[kApplyPer];
        bool live[kApplyPer];
        uint4 ids[kApplyPer][kVecs];
#pragma unroll
        for (int k = 0; k < kApplyPer; ++k) {
            const int64_t j = j0 + threadIdx.x + k * kApplyNT;
            p[k] = j < r.m ? r.apply_pred[j] : -1;
            seen[k] = j < r.m ? r.seen[j] : 0;
            live[k] = p[k] >= 0 && seen[k] >= 0 && seen[k] <= a.n;
            bad |= p[k] >= 0 && !live[k];
            ch[k] = live[k] ? seen[k] / kChunk : a.nch;
            rem[k] = 0;
            if (ch[k] < a.nch) {
                const int64_t sub0 = seen[k] - seen[k] % kSub;   // first entry of the sub-block
                rem[k] = int32_t(seen[k] - sub0);
                const uint4* line =
                    reinterpret_cast<const uint4*>(reinterpret_cast<const char*>(a.w.lb) + sub0 * kIdBytes);
#pragma unroll
                for (int v = 0; v < kVecs; ++v) ids[k][v] = line[v];
            }
        }
#pragma unroll
        for (int k = 0; k < kApplyPer; ++k) {
            const int64_t j = j0 + threadIdx.x + k * kApplyNT;
            if (j >= r.m) continue;
            int32_t q = -1, U = -1;
            if (live[k]) {
                b[k] = win_bucket(ledges, ne, p[k]);
                const int64_t bb = b[k];
                int64_t c = a.w.off[bb * (a.nch + 1) + (ch[k] < a.nch ? ch[k] : a.nch)];
                if (ch[k] < a.nch) {
                    const int sb = int((seen[k] % kChunk) / kSub);
                    c += a.w.t64[(bb * a.nch + ch[k]) * kSubs + sb];
                    // entries of bucket b among the first rem of the sub-block
                    const uint32_t want = uint32_t(bb) * (kByteIds ? 0x01010101u : 0x00010001u);
                    constexpr uint32_t kIdMask = kByteIds ? 0xFFu : 0xFFFFu;
                    int cnt = 0;
#pragma unroll
                    for (int v = 0; v < kVecs; ++v) {
                        const uint32_t w4[4] = {ids[k][v].x, ids[k][v].y, ids[k][v].z, ids[k][v].w};
#pragma unroll
                        for (int h = 0; h < 4; ++h) {
                            const uint32_t x = w4[h] ^ want;   // a zero id field: a match
#pragma unroll
                            for (int f = 0; f < kPerWord; ++f) {
                                const int e = (v * 4 + h) * kPerWord + f;
                                cnt += e < rem[k] && ((x >> (8 * kIdBytes * f)) & kIdMask) == 0u;
                            }
                        }
                    }
                    c += cnt;
                }
                q = a.w.qw[lpbase[bb] + c];
                U = q == MAPS_Q_INF ? r.u_max
                                    : int32_t(int64_t(p[k]) + q < r.u_max ? int64_t(p[k]) + q : r.u_max);
            }
            if (r.q_out) r.q_out[j] = q;
            r.U_out[j] = U;
        }
    }
    if (bad) raise_error(a.dev_err, MAPS_ERR_SEEN_RANGE);
}

}  // namespace
}  // namespace maps

using namespace maps;

extern "C" size_t maps_calibrate_window_workspace_size(int64_t n, int32_t nb) {
    if (n < 0 || nb < 1) return 0;
    return win_carve(nullptr, n, nb).bytes;
}

extern "C" maps_status maps_calibrate_window(const int32_t* pred, const int32_t* truth, int64_t n,
                                             const int32_t* edges, int32_t nb, int32_t window, int32_t alpha_ppm,
                                             const int32_t* apply_pred, const int64_t* apply_seen, int64_t m,
                                             int32_t u_max, int32_t* q_out, int32_t* U_out, uint32_t* dev_err,
                                             void* workspace, size_t workspace_bytes, hipStream_t stream) {
    if (n < 0 || n > INT32_MAX || m < 0 || nb < 1 || nb > MAPS_MAX_WINDOW_BUCKETS || window < 1 ||
        window > MAPS_MAX_WINDOW || u_max < 0)
        return MAPS_E_SIZE;
    if (alpha_ppm <= 0 || alpha_ppm >= 1000000) return MAPS_E_ALPHA;
    if (!dev_err || (n > 0 && (!pred || !truth)) || (nb > 1 && !edges) ||
        (m > 0 && (!apply_pred || !apply_seen || !U_out)) || !workspace)
        return MAPS_E_NULL;
    if (workspace_bytes < maps_calibrate_window_workspace_size(n, nb)) return MAPS_E_WORKSPACE;
    if (m == 0) return MAPS_OK;

    WinArgs a;
    a.pred = pred;
    a.truth = truth;
    a.n = n;
    a.nch = (n + kChunk - 1) / kChunk;
    a.edges = edges;
    a.nb = nb;
    a.window = window;
    a.alpha_ppm = alpha_ppm;
    a.w = win_carve(workspace, n, nb);
    a.dev_err = dev_err;

    if (a.nch > 0) {
        hipLaunchKernelGGL(win_chunk_sort, dim3(unsigned(a.nch)), dim3(kSortNT), 0, stream, a);
        MAPS_CHECK_LAUNCH();
    }
    hipLaunchKernelGGL(win_row_scan, dim3(unsigned(nb)), dim3(256), 0, stream, a);
    MAPS_CHECK_LAUNCH();
    hipLaunchKernelGGL(win_scatter, dim3(unsigned(a.nch > 0 ? a.nch : 1)), dim3(kSortNT), 0, stream, a);
    MAPS_CHECK_LAUNCH();
    // sum_b ceil((n_b + 1) / C) <= (n + nb) / C + nb
    const int64_t groups = (n + nb) / kSelC + nb + 1;
    const SelLayout S = sel_layout(window);
    allow_dynamic_lds(win_select, S.bytes);
    hipLaunchKernelGGL(win_select, dim3(unsigned(groups)), dim3(kSelNT), S.bytes, stream, a);
    MAPS_CHECK_LAUNCH();
    ApplyArgs r{apply_pred, apply_seen, m, u_max, q_out, U_out};
    const int64_t ab = (m + kApplyNT * kApplyPer - 1) / (kApplyNT * kApplyPer);
    const unsigned grid = unsigned(ab < 8192 ? ab : 8192);
    if (nb <= 256) hipLaunchKernelGGL(win_apply<true>, dim3(grid), dim3(kApplyNT), 0, stream, a, r);
    else hipLaunchKernelGGL(win_apply<false>, dim3(grid), dim3(kApplyNT), 0, stream, a, r);
    MAPS_CHECK_LAUNCH();
    return MAPS_OK;
}
