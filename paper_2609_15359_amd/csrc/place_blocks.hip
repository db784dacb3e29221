// Projected placement in blocks of S tokens (Sec. 3.3: KV capacity counted in
// blocks; Eq. (6): a request's blocks are ceil(tokens / S)) on gfx950.
//
// A resident with x = p + g tokens holds ceil((x + t)/S) blocks at step t while
// t <= R.  With x = X S + xi and t = V S + u (0 <= xi, u < S),
//   ceil((x + t)/S) = X + V + [xi + u >= 1] + [xi + u >= S + 1],
// so over the residents still active at t (those with R >= t)
//   OB(t) = sum X + N V + N - [u = 0] #{xi = 0} + #{xi >= S + 1 - u}.
// Per event tau_e (a distinct remaining length) the snapshot keeps N_e,
// sum X and the counts G_e[c] = #{xi >= c} of the residents with R >= tau_e.
// Between events OB and an arrival's ceil((p + t)/S) only grow, so for an
// arrival (p, U), p = P S + rho, with j = #{events < U}:
//   peak = max( P + PMX_rho[j],                      events below U
//               OB(U) + P + ceil((rho + U)/S),         U itself (active set of event j)
//               SMX[first event above U] ),            after U
//   PMX_rho[j] = max_{i < j} (OB(tau_i) + ceil((rho + tau_i)/S)),  SMX[j] = max_{i >= j} OB(tau_i).
//
//   project_blocks   one workgroup per decoder: event bitmap and ranks in LDS,
//                    per-event counters by device atomics in the decoder's
//                    slice, suffix scans, OB at every event, S prefix-max
//                    scans and one suffix-max scan;
//   blocks_order     per tile of 8,192 arrivals: their positions, bounds and
//                    prompts in bound order (a counting sort on 32,768 bound
//                    ranges), so that a wavefront's lanes read the same or
//                    neighbouring events;
//   blocks_pairs     one workgroup per (decoder, tile), the tile in passes of
//                    1,024 pairs, four a thread, each pass's loads issued in
//                    three rounds: every pair's peak from the slice (read
//                    through L2) into the matrix;
//   blocks_finish    per arrival: the choice over the matrix column.
#include "maps_internal.hpp"

namespace maps {
namespace {

constexpr int kPbNT = 1024;
constexpr int kPairsNT = 256;
constexpr int kPairsPer = 4;
constexpr int kOrdNT = 1024;
constexpr int kFinNT = 256;

// Snapshot: a 64-byte header with the arguments it was built for, the decoder
// headers, then the decoder slices.  Placement checks the header against its
// own arguments and each decoder's record count against its seg_off before it
// reads a slice, so a mismatched call raises an error instead of reading past
// the buffer.
constexpr uint32_t kBlkMagic = 0x4250414Du;   // "MAPB"

struct BlkSnapHeader {
    uint32_t magic;
    int32_t D, u_max, S, W, pad0;
    int64_t n_total;
    int32_t pad[8];
};
static_assert(sizeof(BlkSnapHeader) == 64, "block snapshot header size");

// Decoder slice: W rank words {bits, events before}, then per event e = 0..E
// (E+1 records, the last one for "no resident left") the arrays
//   PMX[e][rho] (int32), G[e][c-1] = #{xi >= c} for c = 1..S-1 (int32, rows of
//   Sg = S - 1 rounded up to a multiple of 4), SX[e] (int64), tau[e], N[e],
//   OB[e], SMX[e] (int32; the projection's working arrays when the records do
//   not fit LDS), rec[e] = {tau[e], N[e], SMX[e], SMX[min(e + 1, E)]} (what
//   placement reads of them),
// each with room for capA = n_d + 1 rounded up to a multiple of 4 records.
// PMX starts on a 64-byte boundary and every array is a multiple of 16 bytes
// long, so every array starts 16-byte aligned; when S is a multiple of 4 so
// does every PMX row (the projection writes them 16 bytes at a time), and
// when S is 16 every PMX and G row is one cache line.
struct BlkLayout {
    int32_t D, u_max, S, W;
    int64_t n_total;
    size_t rec;        // bytes per event record slot summed over the arrays
    size_t hdr_bytes;  // decoder headers
    size_t bytes;
};

struct BlkHeader {
    int64_t slice;     // byte offset of the decoder's slice (-1: its seg_off entries were invalid)
    int64_t cap;       // records in the slice: residents + 1
    int32_t E;
    int32_t base;      // max_t OB(t)
};

// Entries per G row: the S - 1 class counts, rounded up to a multiple of 4.
__host__ __device__ inline int64_t blk_gw(int64_t S) { return (S - 1 + 3) & ~int64_t(3); }

__host__ __device__ inline BlkLayout blk_layout(int32_t D, int64_t n_total, int32_t u_max, int32_t S) {
    BlkLayout L;
    L.D = D;
    L.u_max = u_max;
    L.S = S;
    L.W = (((u_max + 1) / 32 + 1) + 1) & ~1;
    L.n_total = n_total;
    // bytes per record, a multiple of 16 so that every slice starts 16-byte aligned
    L.rec = (size_t(4 + 4 + 8 + 4 + 4 + 16) + size_t(blk_gw(S)) * 4 + size_t(S) * 4 + 15) & ~size_t(15);
    L.hdr_bytes = align256(sizeof(BlkSnapHeader) + size_t(D) * sizeof(BlkHeader));
    // slice d starts at hdr + d * (8 W + 4 rec + 64) + seg_off[d] * rec with room for capA <= n_d + 4
    // records after at most 48 bytes of padding
    L.bytes = L.hdr_bytes + size_t(D) * (size_t(L.W) * 8 + 4 * L.rec + 64) + size_t(n_total) * L.rec + 256;
    return L;
}

struct BlkSlice {
    uint2* rank;
    int32_t* tau;
    int32_t* N;
    int64_t* SX;
    int32_t* OB;
    int32_t* SMX;
    int32_t* G;      // [capA][Gw]: class c of event e at G[e * Gw + c]
    int32_t* PMX;    // [capA][S]
    int4* rec;       // [capA]: {tau[e], N[e], SMX[e], SMX[min(e + 1, E)]}, what the pair kernel reads of event e
    int64_t Gw;
};

// Arrays of the slice at byte offset `off` of the snapshot, with room for
// `cap` records (cap = n_d + 1), each array capA = cap rounded up to a
// multiple of 4 entries long.  PMX starts at the next multiple of 64 bytes
// from the snapshot's start, so that with S a multiple of 16 (and the
// snapshot 64-byte aligned, as device allocations are) every PMX and G row
// of 16 entries is one cache line.
__host__ __device__ inline BlkSlice blk_slice(char* snap, int64_t off, const BlkLayout& L, int64_t cap) {
    BlkSlice s;
    const size_t capA = size_t((cap + 3) & ~int64_t(3));
    s.Gw = blk_gw(L.S);
    s.rank = reinterpret_cast<uint2*>(snap + off);
    char* q = snap + ((off + int64_t(L.W) * 8 + 63) & ~int64_t(63));
    s.PMX = reinterpret_cast<int32_t*>(q);
    q += capA * size_t(L.S) * 4;
    s.G = reinterpret_cast<int32_t*>(q);
    q += capA * size_t(s.Gw) * 4;
    s.SX = reinterpret_cast<int64_t*>(q);
    q += capA * 8;
    s.tau = reinterpret_cast<int32_t*>(q);
    q += capA * 4;
    s.N = reinterpret_cast<int32_t*>(q);
    q += capA * 4;
    s.OB = reinterpret_cast<int32_t*>(q);
    q += capA * 4;
    s.SMX = reinterpret_cast<int32_t*>(q);
    q += capA * 4;
    s.rec = reinterpret_cast<int4*>(q);
    return s;
}

__host__ __device__ inline int64_t blk_slice_offset(const BlkLayout& L, int32_t d, int64_t seg_lo) {
    return int64_t(L.hdr_bytes) + int64_t(d) * (int64_t(L.W) * 8 + 4 * int64_t(L.rec) + 64) +
           seg_lo * int64_t(L.rec);
}

__host__ __device__ inline BlkHeader* blk_headers(char* snap) {
    return reinterpret_cast<BlkHeader*>(snap + sizeof(BlkSnapHeader));
}

__device__ inline bool blk_snapshot_ok(const BlkSnapHeader* h, const BlkLayout& L) {
    return h->magic == kBlkMagic && h->D == L.D && h->u_max == L.u_max && h->S == L.S && h->W == L.W &&
           h->n_total == L.n_total;
}

// ceil((r + t) / S) for 0 <= r < S, t >= 0
__device__ inline int64_t ceil_plus(int64_t r, int64_t t, int64_t S) { return (r + t + S - 1) / S; }

// OB at step t from the suffix data of the active set (N, SX, G of the event
// the step lands on); 64-bit.
__device__ inline int64_t occupancy_at(int64_t t, int64_t S, int64_t N, int64_t SX, const int32_t* G) {
    const int64_t V = t / S, u = t % S;
    int64_t ob = SX + N * V + N;
    if (u == 0) ob -= N - (S > 1 ? G[0] : 0);          // #{xi = 0} = N - #{xi >= 1}
    if (u >= 2) ob += G[S - u];                          // #{xi >= S + 1 - u}, stored at c - 1
    return ob;
}

// Quotient and remainder by the block size S for the pair kernel, whose
// operands are below 2^32 (prompts and bounds are 32-bit, residues below S):
// shifts when S is a power of two, else 32-bit division (a 64-bit division
// is a software routine of about a hundred instructions, several per pair).
template <bool kPow2>
struct BlockDiv {
    uint32_t S, sh;
    __device__ uint32_t div(uint32_t n) const {
        if constexpr (kPow2) return n >> sh;
        else return n / S;
    }
    __device__ uint32_t mod(uint32_t n) const {
        if constexpr (kPow2) return n & (S - 1u);
        else return n - div(n) * S;
    }
};

// Phase boundary for the slice in HBM, which only this workgroup touches (one
// CU, one L2): each thread waits until its own stores and atomics have reached
// L2, the barrier, then each thread drops its vector-L1 lines before reading
// what other threads wrote (atomics update L2 only).  No L2 write-back is
// needed, unlike a device-wide fence.
__device__ inline void sync_global() {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
}

// Up to kGroup scans at once over the same len elements (sum or max, forward
// or reverse, inclusive or exclusive), each thread one contiguous chunk:
// get(i, q) and put(i, q, v) for quantity q < nq (kRowPut: put(i, v[kGroup])
// once per element, entries past nq unused).  One pass for the chunk
// totals, one wavefront scan per quantity through DPP, one LDS exchange for
// all of them, one pass to write.  `tmp` holds kGroup * NT / 64 values.
constexpr int kGroup = 16;

template <int NT, bool kMax, bool kReverse, bool kExclusive, typename T, bool kRowPut = false, typename Get,
          typename Put>
__device__ inline void group_scan(int64_t len, int nq, T identity, Get get, Put put, T* tmp) {
    constexpr int kWaves = NT / kWave;
    const int lane = threadIdx.x % kWave, wid = threadIdx.x / kWave;
    const int64_t chunk = (len + NT - 1) / NT;
    const int64_t b = int64_t(threadIdx.x) * chunk;
    const int64_t e = b + chunk < len ? b + chunk : len;
    auto idx = [&](int64_t i) { return kReverse ? len - 1 - i : i; };
    auto op = [](T x, T y) { return kMax ? (x > y ? x : y) : x + y; };
    T acc[kGroup];
#pragma unroll
    for (int q = 0; q < kGroup; ++q) acc[q] = identity;
    for (int64_t i = b; i < e; ++i) {
#pragma unroll
        for (int q = 0; q < kGroup; ++q)
            if (q < nq) acc[q] = op(acc[q], get(idx(i), q));
    }
    __syncthreads();   // tmp may still be read by an earlier scan
#pragma unroll
    for (int q = 0; q < kGroup; ++q) {
        const T incl = kMax ? wave_incl_scan_max(acc[q]) : wave_incl_scan_add(acc[q]);
        if (lane == kWave - 1) tmp[q * kWaves + wid] = incl;
        acc[q] = wave_shift_up1(incl, identity);   // exclusive within the wavefront
    }
    __syncthreads();
    if constexpr (kWaves == 16) {
        // every quantity's prefix over the wavefronts at once: thread (q, w) of the first kGroup
        // wavefront-rows holds tmp[q][w], one DPP row of 16 lanes scans it, and the row shifted by one
        // is the exclusive prefix (each thread rewrites only its own entry)
        if (threadIdx.x < kGroup * kWaves) {
            T incl = tmp[threadIdx.x];
            incl = op(incl, dpp_move<kDppRowShr1, 0xf>(identity, incl));
            incl = op(incl, dpp_move<kDppRowShr2, 0xf>(identity, incl));
            incl = op(incl, dpp_move<kDppRowShr4, 0xf>(identity, incl));
            incl = op(incl, dpp_move<kDppRowShr8, 0xf>(identity, incl));
            tmp[threadIdx.x] = dpp_move<kDppRowShr1, 0xf>(identity, incl);
        }
        __syncthreads();
#pragma unroll
        for (int q = 0; q < kGroup; ++q) acc[q] = op(tmp[q * kWaves + wid], acc[q]);
    } else {
#pragma unroll
        for (int q = 0; q < kGroup; ++q) {
            T before = identity;
            for (int w = 0; w < wid; ++w) before = op(before, tmp[q * kWaves + w]);
            acc[q] = op(before, acc[q]);
        }
    }
    for (int64_t i = b; i < e; ++i) {
        T out[kGroup];
#pragma unroll
        for (int q = 0; q < kGroup; ++q) {
            out[q] = identity;
            if (q < nq) {
                const T x = get(idx(i), q);
                const T next = op(acc[q], x);
                out[q] = kExclusive ? acc[q] : next;
                if constexpr (!kRowPut) put(idx(i), q, out[q]);
                acc[q] = next;
            }
        }
        if constexpr (kRowPut) put(idx(i), out);   // all nq results of element i at once
    }
    __syncthreads();
}

struct ProjArgs {
    BlkLayout L;
    const int64_t* seg_off;
    const int32_t* p;
    const int32_t* g;
    const int32_t* U;
    char* snap;
    int32_t* base_peak;
    uint32_t* dev_err;
    int64_t lds_cap;   // event records that fit the LDS arrays past the bitmap (0: every decoder in HBM)
};

// The per-event arrays of one decoder in LDS (past the W bitmap words and the
// W rank counts), every count of a record summed with LDS atomics, the scans
// done in LDS, and the slice written to HBM once at the end.
struct LdsRecs {
    uint32_t* tau;
    uint32_t* N;
    unsigned long long* SX;
    int32_t* OB;
    uint32_t* G;   // [cap][Gw]: class c (c = 0..S-2, for xi = c + 1) in half (c & 1) of word c / 2
    int64_t Gw;
    __device__ uint32_t g(int64_t e, int c) const { return (G[e * Gw + c / 2] >> (16 * (c & 1))) & 0xFFFFu; }
    __device__ void set_g(int64_t e, int c, uint32_t v) const {
        uint32_t& w = G[e * Gw + c / 2];
        const int sh = 16 * (c & 1);
        w = (w & ~(0xFFFFu << sh)) | (v << sh);
    }
};

// The 16-bit class counts hold because a decoder on this path has fewer than
// 65,536 residents: no count, sum of counts or suffix sum reaches 2^16.
__device__ __forceinline__ void project_blocks_lds(const ProjArgs& a, int d, int64_t lo, int64_t hi, uint32_t E,
                                                   const uint32_t* bits, const uint32_t* wpre, const BlkSlice& s,
                                                   int64_t off, int64_t cap, int64_t* red64, uint32_t* red32,
                                                   int32_t* redg) {
    const BlkLayout& L = a.L;
    const int tid = threadIdx.x;
    const int64_t S = L.S;
    const int64_t len = int64_t(E) + 1;   // the events and the record past the last one
    LdsRecs r;
    uint32_t* base = const_cast<uint32_t*>(wpre) + L.W;
    r.Gw = S / 2;   // ceil((S - 1) / 2) halves
    r.tau = base;
    r.N = r.tau + len;
    r.SX = reinterpret_cast<unsigned long long*>(r.N + len);   // 8-byte aligned: 8 W + 8 len bytes in
    r.OB = reinterpret_cast<int32_t*>(r.SX + len);
    r.G = reinterpret_cast<uint32_t*>(r.OB + len);
    // 3'. event times; counters zeroed
    for (int64_t e = tid; e < len; e += kPbNT) {
        r.tau[e] = 0;
        r.N[e] = 0;
        r.SX[e] = 0;
        for (int64_t c = 0; c < r.Gw; ++c) r.G[e * r.Gw + c] = 0;
    }
    __syncthreads();
    for (int w = tid; w < L.W; w += kPbNT) {
        uint32_t b = bits[w], e = wpre[w];
        while (b) {
            r.tau[e++] = uint32_t(w * 32 + (__ffs(b) - 1));
            b &= b - 1u;
        }
    }
    // each resident adds itself to its event: 1, X = x div S, and its class xi = x mod S
    for (int64_t i = lo + tid; i < hi; i += kPbNT) {
        int32_t pr = a.p[i], gr = a.g[i], ur = a.U[i];
        pr = pr < 0 ? 0 : pr;
        gr = gr < 0 ? 0 : gr;
        ur = ur < 0 ? 0 : ur;
        int64_t R = int64_t(ur) - gr;
        R = R > 0 ? R : 0;
        R = R > L.u_max ? L.u_max : R;
        const uint32_t e = wpre[R >> 5] + __popc(bits[R >> 5] & ((1u << (R & 31)) - 1u));
        const int64_t x = int64_t(pr) + gr;
        atomicAdd(&r.N[e], 1u);
        atomicAdd(&r.SX[e], (unsigned long long)(x / S));
        const int xi = int(x % S);
        if (xi >= 1) atomicAdd(&r.G[e * r.Gw + (xi - 1) / 2], ((xi - 1) & 1) ? 0x10000u : 1u);
    }
    __syncthreads();
    // 4'. suffix sums over the events (record E is zero): SX, then N and every class count
    block_scan<kPbNT, false, true, false, int64_t>(
        len, int64_t(0), [&](int64_t e) { return int64_t(r.SX[e]); },
        [&](int64_t e, int64_t v) { r.SX[e] = (unsigned long long)v; }, red64);
    for (int q0 = 0; q0 < S; q0 += kGroup)
        group_scan<kPbNT, false, true, false, int32_t>(
            len, int(S - q0 < kGroup ? S - q0 : kGroup), 0,
            [&](int64_t e, int q) { return q0 + q == 0 ? int32_t(r.N[e]) : int32_t(r.g(e, q0 + q - 1)); },
            [&](int64_t e, int q, int32_t v) {
                if (q0 + q == 0) r.N[e] = uint32_t(v);
                else r.set_g(e, q0 + q - 1, uint32_t(v));
            },
            redg);   // ends with a barrier
    // counts by class -> counts of classes >= c, and the occupancy at every event
    bool big = false;
    for (int64_t e = tid; e < len; e += kPbNT) {
        uint32_t acc = 0;
        for (int c = int(S) - 2; c >= 0; --c) {
            acc += r.g(e, c);
            r.set_g(e, c, acc);
        }
        int64_t ob = 0;
        if (e < int64_t(E)) {
            // occupancy_at with the class counts read from the halves
            const int64_t t = r.tau[e], V = t / S, u = t % S, N = r.N[e];
            ob = int64_t(r.SX[e]) + N * V + N;
            if (u == 0) ob -= N - (S > 1 ? int64_t(r.g(e, 0)) : 0);
            if (u >= 2) ob += r.g(e, int(S - u));   // #{xi >= S + 1 - u}: class S - u
        }
        big |= ob + 2 * int64_t(L.u_max) / S + 2 > int64_t(INT32_MAX) / 2;
        r.OB[e] = int32_t(ob > INT32_MAX ? INT32_MAX : ob);
    }
    if (big) raise_error(a.dev_err, MAPS_ERR_INT32_RANGE);
    __syncthreads();
    // 6'. prefix maxima per residue class (exclusive: events below) into the
    // slice, the suffix maximum, then the slice's event arrays
    // with S a multiple of 4 every row, and every group of kGroup residues in it, starts 16-byte aligned
    const bool vec = S % 4 == 0 && (reinterpret_cast<uintptr_t>(s.PMX) & 15) == 0;
    for (int r0 = 0; r0 < S; r0 += kGroup) {
        const int nq = int(S - r0 < kGroup ? S - r0 : kGroup);
        group_scan<kPbNT, true, false, true, int32_t, true>(
            len, nq, 0,
            [&](int64_t e, int q) {
                return e < int64_t(E) ? int32_t(r.OB[e] + ceil_plus(r0 + q, r.tau[e], S)) : 0;
            },
            [&](int64_t e, const int32_t (&v)[kGroup]) {
                int32_t* dst = s.PMX + e * S + r0;
                if (vec) {
#pragma unroll
                    for (int q = 0; q < kGroup; q += 4)
                        if (q < nq) *reinterpret_cast<int4*>(dst + q) = make_int4(v[q], v[q + 1], v[q + 2], v[q + 3]);
                } else {
#pragma unroll
                    for (int q = 0; q < kGroup; ++q)
                        if (q < nq) dst[q] = v[q];
                }
            },
            redg);
    }
    // placement reads SX and the event records; tau, N, OB and the suffix maxima as arrays of their own are
    // the HBM path's working copies and are not written here
    for (int64_t e = tid; e < len; e += kPbNT) s.SX[e] = int64_t(r.SX[e]);
    __syncthreads();   // SX is out: its LDS array takes the suffix maxima
    int32_t* smx = reinterpret_cast<int32_t*>(r.SX);
    const int32_t base_pk = block_scan<kPbNT, true, true, false, int32_t>(
        len, 0, [&](int64_t e) { return r.OB[e]; }, [&](int64_t e, int32_t v) { smx[e] = v; },
        reinterpret_cast<int32_t*>(red32));   // ends with a barrier
    // the pair kernel's record of every event
    for (int64_t e = tid; e < len; e += kPbNT)
        s.rec[e] = make_int4(e < int64_t(E) ? int32_t(r.tau[e]) : 0, int32_t(r.N[e]), smx[e],
                             smx[e + 1 < len ? e + 1 : e]);
    // the class rows in address order, Gw entries an event (the padding past S - 1 classes zero): each
    // wavefront stores whole lines (len Gw is below 2^31 here: fewer than 65,536 records)
    const uint32_t gw = uint32_t(s.Gw);
    for (uint32_t k = tid; k < uint32_t(len) * gw; k += kPbNT) {
        const uint32_t e = k / gw, c = k - e * gw;
        s.G[k] = c + 1 < uint32_t(S) ? int32_t(r.g(e, int(c))) : 0;
    }
    if (tid == 0) {
        BlkHeader* hdr = blk_headers(a.snap);
        hdr[d].slice = off;
        hdr[d].cap = cap;
        hdr[d].E = int32_t(E);
        hdr[d].base = base_pk;
        a.base_peak[d] = base_pk;
    }
}

__global__ __launch_bounds__(kPbNT) void project_blocks(ProjArgs a) {
    extern __shared__ uint32_t bits[];               // W bit words, then W counts of events before each
    __shared__ int64_t red64[kPbNT / kWave];
    __shared__ uint32_t red32[kPbNT / kWave];
    __shared__ int32_t redg[kGroup * (kPbNT / kWave)];
    const BlkLayout& L = a.L;
    uint32_t* wpre = bits + L.W;
    const int d = blockIdx.x;
    const int tid = threadIdx.x;
    const int64_t lo = a.seg_off[d], hi = a.seg_off[d + 1];
    BlkHeader* hdr = blk_headers(a.snap);
    if (d == 0 && tid == 0) {   // every field is known before the decoders
        BlkSnapHeader h;
        h.D = L.D;
        h.u_max = L.u_max;
        h.S = L.S;
        h.W = L.W;
        h.pad0 = 0;
        h.n_total = L.n_total;
        for (int i = 0; i < 8; ++i) h.pad[i] = 0;
        h.magic = kBlkMagic;
        *reinterpret_cast<BlkSnapHeader*>(a.snap) = h;
    }
    if (!(0 <= lo && lo <= hi && hi <= L.n_total)) {
        if (tid == 0) {
            raise_error(a.dev_err, MAPS_ERR_SEG_OFFSETS);
            hdr[d].E = 0;
            hdr[d].base = 0;
            hdr[d].slice = -1;
            hdr[d].cap = 0;
            a.base_peak[d] = 0;
        }
        return;
    }
    const int64_t n = hi - lo, cap = n + 1;
    const int64_t S = L.S;
    const int64_t off = blk_slice_offset(L, d, lo);
    BlkSlice s = blk_slice(a.snap, off, L, cap);

    // 1. event bitmap over the step axis
    for (int w = tid; w < L.W; w += kPbNT) bits[w] = 0u;
    __syncthreads();
    bool neg = false, range = false;
    for (int64_t r = lo + tid; r < hi; r += kPbNT) {
        int32_t pr = a.p[r], gr = a.g[r], ur = a.U[r];
        neg |= (pr < 0) | (gr < 0) | (ur < 0);
        gr = gr < 0 ? 0 : gr;
        ur = ur < 0 ? 0 : ur;
        int64_t R = int64_t(ur) - gr;
        R = R > 0 ? R : 0;
        if (R > L.u_max) { range = true; R = L.u_max; }
        atomicOr(&bits[R >> 5], 1u << (R & 31));
    }
    if (neg) raise_error(a.dev_err, MAPS_ERR_NEG_LEN);
    if (range) raise_error(a.dev_err, MAPS_ERR_BOUND_RANGE);
    __syncthreads();

    // 2. ranks: events before each word; the rank words and event times
    const uint32_t E = block_scan<kPbNT, false, false, true, uint32_t>(
        L.W, 0u, [&](int64_t w) { return uint32_t(__popc(bits[w])); },
        [&](int64_t w, uint32_t v) {
            wpre[w] = v;
            s.rank[w] = make_uint2(bits[w], v);
        },
        red32);
    if (int64_t(E) + 1 <= a.lds_cap && n < 65536) {   // the same in every thread
        project_blocks_lds(a, d, lo, hi, E, bits, wpre, s, off, cap, red64, red32, redg);
        return;
    }
    for (int w = tid; w < L.W; w += kPbNT) {
        uint32_t b = bits[w], e = wpre[w];
        while (b) {
            s.tau[e++] = int32_t(w * 32 + (__ffs(b) - 1));
            b &= b - 1u;
        }
    }
    // counters of every record (the one past the last event stays zero)
    for (int64_t e = tid; e <= int64_t(E); e += kPbNT) {
        s.N[e] = 0;
        s.SX[e] = 0;
        for (int c = 0; c + 1 < S; ++c) s.G[e * s.Gw + c] = 0;
    }
    sync_global();

    // 3. each resident adds itself to its event: 1, X = x div S, and its class xi = x mod S
    for (int64_t r = lo + tid; r < hi; r += kPbNT) {
        int32_t pr = a.p[r], gr = a.g[r], ur = a.U[r];
        pr = pr < 0 ? 0 : pr;
        gr = gr < 0 ? 0 : gr;
        ur = ur < 0 ? 0 : ur;
        int64_t R = int64_t(ur) - gr;
        R = R > 0 ? R : 0;
        R = R > L.u_max ? L.u_max : R;
        const uint32_t e = wpre[R >> 5] + __popc(bits[R >> 5] & ((1u << (R & 31)) - 1u));
        const int64_t x = int64_t(pr) + gr;
        atomicAdd(&s.N[e], 1);
        atomicAdd(reinterpret_cast<unsigned long long*>(&s.SX[e]), (unsigned long long)(x / S));
        const int xi = int(x % S);
        if (xi >= 1) atomicAdd(&s.G[e * s.Gw + (xi - 1)], 1);
    }
    sync_global();

    // 4. suffix sums over the events (record E is zero): N, SX and every class count
    const int64_t len = int64_t(E) + 1;
    block_scan<kPbNT, false, true, false, int64_t>(
        len, int64_t(0), [&](int64_t e) { return s.SX[e]; }, [&](int64_t e, int64_t v) { s.SX[e] = v; }, red64);
    // N (quantity 0) and the S - 1 class counts (quantity c), kGroup at a time
    for (int q0 = 0; q0 < S; q0 += kGroup) {
        auto cell = [&](int64_t e, int q) -> int32_t& {
            return q0 + q == 0 ? s.N[e] : s.G[e * s.Gw + (q0 + q - 1)];
        };
        group_scan<kPbNT, false, true, false, int32_t>(
            len, int(S - q0 < kGroup ? S - q0 : kGroup), 0, [&](int64_t e, int q) { return cell(e, q); },
            [&](int64_t e, int q, int32_t v) { cell(e, q) = v; }, redg);
    }
    sync_global();
    // counts by class -> counts of classes >= c
    for (int64_t e = tid; e < len; e += kPbNT) {
        int32_t acc = 0;
        for (int c = int(S) - 2; c >= 0; --c) {
            acc += s.G[e * s.Gw + c];
            s.G[e * s.Gw + c] = acc;
        }
    }
    sync_global();

    // 5. occupancy at every event (record E: nobody left)
    bool big = false;
    for (int64_t e = tid; e < len; e += kPbNT) {
        int64_t ob = 0;
        if (e < int64_t(E)) ob = occupancy_at(s.tau[e], S, s.N[e], s.SX[e], s.G + e * s.Gw);
        big |= ob + 2 * int64_t(L.u_max) / S + 2 > int64_t(INT32_MAX) / 2;
        s.OB[e] = int32_t(ob > INT32_MAX ? INT32_MAX : ob);
    }
    if (big) raise_error(a.dev_err, MAPS_ERR_INT32_RANGE);
    sync_global();

    // 6. prefix maxima per residue class (exclusive: events below), suffix maximum
    for (int r0 = 0; r0 < S; r0 += kGroup)
        group_scan<kPbNT, true, false, true, int32_t>(
            len, int(S - r0 < kGroup ? S - r0 : kGroup), 0,
            [&](int64_t e, int q) {
                return e < int64_t(E) ? int32_t(s.OB[e] + ceil_plus(r0 + q, s.tau[e], S)) : 0;
            },
            [&](int64_t e, int q, int32_t v) { s.PMX[e * S + r0 + q] = v; }, redg);
    const int32_t base = block_scan<kPbNT, true, true, false, int32_t>(
        len, 0, [&](int64_t e) { return s.OB[e]; }, [&](int64_t e, int32_t v) { s.SMX[e] = v; },
        reinterpret_cast<int32_t*>(red32));
    sync_global();
    for (int64_t e = tid; e < len; e += kPbNT)
        s.rec[e] = make_int4(e < int64_t(E) ? s.tau[e] : 0, s.N[e], s.SMX[e], s.SMX[e + 1 < len ? e + 1 : e]);
    if (tid == 0) {
        hdr[d].slice = off;
        hdr[d].cap = cap;
        hdr[d].E = int32_t(E);
        hdr[d].base = base;
        a.base_peak[d] = base;
    }
}

struct PairArgs {
    BlkLayout L;
    const char* snap;
    const int32_t* ap;
    const int32_t* aU;
    int64_t A;
    const int64_t* seg_off;
    int32_t* pair;
    int32_t* order;   // per tile of kTile arrivals: their tile indices, by bound
    int32_t* sU;      // the same tile's bounds in that order
    int32_t* sp;      // and prompts
    uint32_t* dev_err;
};

// A tile of kTile arrivals is sorted by bound once; each decoder's workgroup
// takes it in passes of kPass pairs, kPairsPer per thread.  The larger the
// tile, the fewer distinct events the 64 sorted arrivals of a wavefront land
// on, so the fewer cache lines each of the pair kernel's loads touches.
constexpr int kPass = kPairsNT * kPairsPer;
constexpr int kTile = 8192;
constexpr int kOrdPer = kTile / kOrdNT;
constexpr int kOrdBins = 32768;   // bound ranges of the counting sort, a power of two
static_assert(kTile % kPass == 0 && kTile % kOrdNT == 0, "whole passes and order rounds per tile");
static_assert(kOrdBins % kOrdNT == 0, "whole rounds of 64 bins per wavefront in the scan");

// The arrivals of each tile ordered by their bound (a counting sort on
// kOrdBins bound ranges of 2^sh steps, sh the least that covers 0..u_max), so
// that the lanes of a wavefront read neighbouring events of a decoder's slice.
// Written once, used by every decoder's workgroup.
__global__ __launch_bounds__(kOrdNT) void blocks_order(PairArgs a) {
    __shared__ int32_t start[kOrdBins];
    __shared__ int32_t tmp[kOrdNT / kWave];
    const int64_t base = int64_t(blockIdx.x) * kTile;
    const int64_t left = a.A - base;
    const int n = left < kTile ? int(left) : kTile;
    for (int b = threadIdx.x; b < kOrdBins; b += kOrdNT) start[b] = 0;
    int32_t Uv[kOrdPer], pv[kOrdPer];
#pragma unroll
    for (int k = 0; k < kOrdPer; ++k) {
        const int t = threadIdx.x + k * kOrdNT;
        Uv[k] = t < n ? a.aU[base + t] : 0;
        pv[k] = t < n ? a.ap[base + t] : 0;
    }
    const int32_t top = a.L.u_max;   // bounds above u_max share the last range
    int sh = 0;
    while ((top >> sh) >= kOrdBins) ++sh;
    __syncthreads();
    int key[kOrdPer];
#pragma unroll
    for (int k = 0; k < kOrdPer; ++k) {
        const int t = threadIdx.x + k * kOrdNT;
        const int32_t u = Uv[k] < 0 ? 0 : (Uv[k] < top ? Uv[k] : top);
        key[k] = u >> sh;
        if (t < n) atomicAdd(&start[key[k]], 1);
    }
    __syncthreads();
    {
        // exclusive prefix over the bins: wavefront w takes the contiguous bins [w kSeg, (w + 1) kSeg), 64 at a
        // time (lane l reads bin 64 r + l of round r, so no two lanes share an LDS bank), once for its total
        // and, after the totals are exchanged, once more for the prefix
        constexpr int kWaves = kOrdNT / kWave;
        constexpr int kSeg = kOrdBins / kWaves;
        const int lane = threadIdx.x % kWave, wid = threadIdx.x / kWave;
        int32_t* seg = start + wid * kSeg;
        int32_t part = 0;
        for (int r = 0; r < kSeg; r += kWave) part += seg[r + lane];
        part = wave_reduce_add(part);
        if (lane == 0) tmp[wid] = part;
        __syncthreads();
        int32_t carry = 0;
#pragma unroll
        for (int w = 0; w < kWaves; ++w)
            if (w < wid) carry += tmp[w];
        for (int r = 0; r < kSeg; r += kWave) {
            const int32_t v = seg[r + lane];
            const int32_t incl = wave_incl_scan_add(v);
            seg[r + lane] = carry + incl - v;
            carry += wave_last(incl);
        }
        __syncthreads();
    }
#pragma unroll
    for (int k = 0; k < kOrdPer; ++k) {
        const int t = threadIdx.x + k * kOrdNT;
        if (t < n) {
            const int64_t o = base + atomicAdd(&start[key[k]], 1);
            a.order[o] = t;
            a.sU[o] = Uv[k];
            a.sp[o] = pv[k];
        }
    }
}

// Every pair's peak in blocks; the tile's arrivals taken in bound order, the
// row of the matrix written back in arrival order from LDS.  One workgroup
// per (decoder, tile), numbered so that the workgroups of one decoder are
// consecutive among those of one XCD (workgroup b runs on XCD b mod 8): XCD x
// takes decoders x, x + 8, ... one after another, every tile of a decoder
// while its slice is in that XCD's L2, instead of each of the 8 L2s fetching
// every slice.
constexpr int kXcds = 8;
template <bool kPow2>
__global__ __launch_bounds__(kPairsNT) void blocks_pairs(PairArgs a, int64_t tiles) {
    __shared__ int32_t row[kTile];
    const BlkLayout& L = a.L;
    const int64_t k = int64_t(blockIdx.x) / kXcds;   // the k-th workgroup of its XCD
    const int d = int(blockIdx.x % kXcds) + kXcds * int(k / tiles);
    const int64_t tile = k % tiles;
    if (d >= L.D) return;   // the last round of decoders when D is not a multiple of 8
    if (!blk_snapshot_ok(reinterpret_cast<const BlkSnapHeader*>(a.snap), L)) {
        if (tile == 0 && d == 0 && threadIdx.x == 0) raise_error(a.dev_err, MAPS_ERR_SNAPSHOT);
        return;
    }
    const BlkHeader h = blk_headers(const_cast<char*>(a.snap))[d];
    const int64_t S = L.S;
    const int64_t base = tile * kTile;
    const int64_t left = a.A - base;
    const int n = left < kTile ? int(left) : kTile;
    const int64_t cap = a.seg_off[d + 1] - a.seg_off[d] + 1;
    if (h.slice < 0 || h.cap != cap) {
        if (h.slice >= 0 && tile == 0 && threadIdx.x == 0) raise_error(a.dev_err, MAPS_ERR_SNAPSHOT);
        for (int t = threadIdx.x; t < n; t += kPairsNT) a.pair[int64_t(d) * a.A + base + t] = -1;
        return;
    }
    BlkSlice s = blk_slice(const_cast<char*>(a.snap), h.slice, L, cap);
    const int32_t E = h.E;
    const int32_t tmax = 32 * L.W - 1;
    const BlockDiv<kPow2> dv{uint32_t(S), uint32_t(__builtin_ctzll(uint64_t(S)))};
    // The kPairsPer pairs of a thread go through three rounds of loads together:
    // the tile's (position, bound, prompt) in bound order, the rank words, then
    // the event's entries; a pair without a bound (or past the tile) reads event 0
    // and is written as -1.
    bool neg = false, big = false;
    for (int p0 = 0; p0 < n; p0 += kPass) {
        int32_t loc[kPairsPer], Uv[kPairsPer], pv[kPairsPer];
#pragma unroll
        for (int k = 0; k < kPairsPer; ++k) {
            const int t = p0 + threadIdx.x + k * kPairsNT;
            const bool in = t < n;
            loc[k] = in ? a.order[base + t] : -1;
            Uv[k] = in ? a.sU[base + t] : -1;
            pv[k] = in ? a.sp[base + t] : 0;
        }
        uint2 w[kPairsPer];
#pragma unroll
        for (int k = 0; k < kPairsPer; ++k) {
            const int32_t tc = Uv[k] < 0 ? 0 : (Uv[k] < tmax ? Uv[k] : tmax);
            w[k] = s.rank[tc >> 5];
        }
        int32_t pmx[kPairsPer], nj[kPairsPer], gj[kPairsPer], tj[kPairsPer], sm0[kPairsPer], sm1[kPairsPer];
        int64_t sx[kPairsPer];
        int32_t jj[kPairsPer];
#pragma unroll
        for (int k = 0; k < kPairsPer; ++k) {
            const int32_t U = Uv[k] < 0 ? 0 : Uv[k];
            const int32_t tc = U < tmax ? U : tmax;
            int32_t j = int32_t(w[k].y) + __popc(w[k].x & ((1u << (tc & 31)) - 1u));
            j = j < E ? j : E;
            jj[k] = j;
            const uint32_t p = uint32_t(pv[k] < 0 ? 0 : pv[k]);
            const uint32_t u = dv.mod(uint32_t(U));
            // G index: Gj[0] when u = 0, Gj[S - u] when u >= 2, unused otherwise (read at 0)
            const int64_t gi = u >= 2 ? int64_t(S) - u : 0;
            const int32_t jr = j < E ? j : 0;   // the entries of a real event; E has none
            pmx[k] = s.PMX[int64_t(j) * S + dv.mod(p)];
            const int4 rc = s.rec[j];   // tau, N, SMX(j), SMX(j + 1) of event j: one 16-byte load
            nj[k] = rc.y;
            gj[k] = S > 1 ? s.G[int64_t(jr) * s.Gw + gi] : 0;
            sx[k] = s.SX[jr];
            tj[k] = rc.x;
            sm0[k] = rc.z;
            sm1[k] = rc.w;
        }
#pragma unroll
        for (int k = 0; k < kPairsPer; ++k) {
            if (loc[k] < 0) continue;
            const int32_t U = Uv[k];
            int32_t out = -1;
            if (U >= 0) {
                neg |= pv[k] < 0;
                const int64_t p = pv[k] < 0 ? 0 : pv[k];
                const int32_t j = jj[k];
                const int64_t P = dv.div(uint32_t(p)), rho = dv.mod(uint32_t(p));
                const int64_t left = P + pmx[k];
                int64_t at = P + dv.div(uint32_t(rho + U + S - 1));   // ceil((rho + U) / S)
                if (j < E) {
                    // occupancy at U (as occupancy_at, with the quotient and remainder of U taken here)
                    const int64_t V = dv.div(uint32_t(U)), u = dv.mod(uint32_t(U)), N = nj[k];
                    int64_t ob = sx[k] + N * V + N;
                    if (u == 0) ob -= N - gj[k];
                    if (u >= 2) ob += gj[k];
                    at += ob;
                }
                const int64_t after = (j < E && tj[k] == U) ? sm1[k] : sm0[k];
                int64_t pk = left > at ? left : at;
                pk = pk > after ? pk : after;
                big |= pk > INT32_MAX;
                out = int32_t(pk > INT32_MAX ? INT32_MAX : pk);
            }
            row[loc[k]] = out;
        }
    }
    // a negative prompt, or a peak clamped to INT32_MAX, is reported once per wavefront
    if (__builtin_amdgcn_ballot_w64(neg) != 0 && threadIdx.x % kWave == 0) raise_error(a.dev_err, MAPS_ERR_NEG_LEN);
    if (__builtin_amdgcn_ballot_w64(big) != 0 && threadIdx.x % kWave == 0)
        raise_error(a.dev_err, MAPS_ERR_INT32_RANGE);
    __syncthreads();
    // non-temporal stores: the matrix rows stream past L2 instead of evicting the decoder slices that the
    // same XCD's other workgroups still read (measured 9% faster here; the token path's row stores are
    // the other way round)
    for (int t = threadIdx.x; t < n; t += kPairsNT)
        __builtin_nontemporal_store(row[t], &a.pair[int64_t(d) * a.A + base + t]);
}

struct FinArgs {
    uint32_t* dev_err;
    int32_t D;
    int32_t S;
    const int32_t* cap;
    const int32_t* qlen;
    const int32_t* aU;
    int64_t A;
    int32_t policy;
    int64_t rr_offset;
    const int32_t* pair;
    int32_t* choice;
    int32_t* chosen_peak;
    int32_t* chosen_overflow;
    uint8_t* flags;
};

// Algorithm 1's choice per arrival over its column of the matrix.  Capacities
// in blocks and queue lengths are staged in LDS, kFinDec decoders at a time,
// and each thread keeps kFinUnroll column loads in flight; the decoders are
// still taken in index order, so ties go to the lowest index as before.
constexpr int kFinDec = 1024;
constexpr int kFinUnroll = 16;

__global__ __launch_bounds__(kFinNT) void blocks_finish(FinArgs a) {
    __shared__ int32_t lcap[kFinDec];   // floor(capacity / S)
    __shared__ int32_t lq[kFinDec];
    const int64_t stride = int64_t(gridDim.x) * kFinNT;
    // every thread runs the same number of rounds: the staging barriers are block-wide
    for (int64_t i0 = int64_t(blockIdx.x) * kFinNT; i0 < a.A; i0 += stride) {
        const int64_t i = i0 + threadIdx.x;
        const bool live = i < a.A;
        const int32_t U = live ? a.aU[i] : -1;
        int32_t feas = -1, fq = 0, fpk = 0, fb = -1, fbpk = 0;
        int64_t fbslack = 0;
        auto consider = [&](int32_t d, int32_t pk, int32_t capb, int32_t q) {
            const int64_t slack = int64_t(capb) - pk;
            if (a.policy == MAPS_POLICY_MQ && slack >= 0 && (feas < 0 || q < fq)) {
                feas = d;
                fq = q;
                fpk = pk;
            }
            if (fb < 0 || slack > fbslack) {
                fb = d;
                fbslack = slack;
                fbpk = pk;
            }
        };
        for (int32_t d0 = 0; d0 < a.D; d0 += kFinDec) {
            const int32_t nd = a.D - d0 < kFinDec ? a.D - d0 : kFinDec;
            __syncthreads();
            for (int k = threadIdx.x; k < nd; k += kFinNT) {
                const int32_t c = a.cap[d0 + k], q = a.qlen[d0 + k];
                // a negative capacity or queue length is an error (its block count would
                // truncate toward zero); each workgroup checks every decoder, the first reports
                if ((c < 0 || q < 0) && blockIdx.x == 0) raise_error(a.dev_err, MAPS_ERR_NEG_LEN);
                lcap[k] = c < 0 ? -1 : c / a.S;
                lq[k] = q;
            }
            __syncthreads();
            if (!live || U < 0) continue;
            const int32_t* col = a.pair + int64_t(d0) * a.A + i;
            int k = 0;
            for (; k + kFinUnroll <= nd; k += kFinUnroll) {
                int32_t pk[kFinUnroll];
#pragma unroll
                for (int u = 0; u < kFinUnroll; ++u) pk[u] = col[int64_t(k + u) * a.A];
#pragma unroll
                for (int u = 0; u < kFinUnroll; ++u) consider(d0 + k + u, pk[u], lcap[k + u], lq[k + u]);
            }
            for (; k < nd; ++k) consider(d0 + k, col[int64_t(k) * a.A], lcap[k], lq[k]);
        }
        if (!live) continue;
        if (U < 0) {
            a.choice[i] = int32_t((a.rr_offset + i) % a.D);
            a.chosen_peak[i] = -1;
            a.chosen_overflow[i] = 0;
            a.flags[i] = 2;
        } else if (feas >= 0) {
            a.choice[i] = feas;
            a.chosen_peak[i] = fpk;
            a.chosen_overflow[i] = 0;
            a.flags[i] = 1;
        } else {
            a.choice[i] = fb;
            a.chosen_peak[i] = fbpk;
            a.chosen_overflow[i] = fbslack < 0 ? int32_t(-fbslack) : 0;
            a.flags[i] = fbslack >= 0 ? 1 : 0;
        }
    }
}

}  // namespace
}  // namespace maps

using namespace maps;

extern "C" size_t maps_blocks_snapshot_bytes(int32_t D, int64_t n_total, int32_t u_max, int32_t block_size) {
    if (D < 1 || n_total < 0 || u_max < 0 || u_max > MAPS_MAX_BLOCKS_U_MAX || block_size < 1 ||
        block_size > MAPS_MAX_BLOCK_SIZE)
        return 0;
    return blk_layout(D, n_total, u_max, block_size).bytes;
}

extern "C" maps_status maps_project_blocks(int32_t D, const int64_t* seg_off, const int32_t* prompt,
                                           const int32_t* generated, const int32_t* upper, int64_t n_total,
                                           int32_t u_max, int32_t block_size, void* snapshot,
                                           size_t snapshot_bytes, int32_t* base_peak, uint32_t* dev_err,
                                           hipStream_t stream) {
    if (D < 1 || n_total < 0 || u_max < 0 || u_max > MAPS_MAX_BLOCKS_U_MAX || block_size < 1 ||
        block_size > MAPS_MAX_BLOCK_SIZE)
        return MAPS_E_SIZE;
    if (!seg_off || !snapshot || !base_peak || !dev_err || (n_total > 0 && (!prompt || !generated || !upper)))
        return MAPS_E_NULL;
    const BlkLayout L = blk_layout(D, n_total, u_max, block_size);
    if (snapshot_bytes < L.bytes) return MAPS_E_BUFFER;
    // the bitmap and its rank counts, then as many LDS event records as fit 152 KB
    const size_t fixed = size_t(L.W) * 8;
    const size_t per_rec = size_t(4 + 4 + 8 + 4) + size_t(block_size / 2) * 4;
    constexpr size_t kBudget = 152 * 1024;
    int64_t lds_cap = fixed + 64 < kBudget ? int64_t((kBudget - fixed - 64) / per_rec) : 0;
    ProjArgs a{L, seg_off, prompt, generated, upper, static_cast<char*>(snapshot), base_peak, dev_err, lds_cap};
    const size_t lds = fixed + (lds_cap > 0 ? size_t(lds_cap) * per_rec + 64 : 0);
    allow_dynamic_lds(project_blocks, lds);
    hipLaunchKernelGGL(project_blocks, dim3(unsigned(D)), dim3(kPbNT), lds, stream, a);
    MAPS_CHECK_LAUNCH();
    return MAPS_OK;
}

extern "C" maps_status maps_place_blocks(const void* snapshot, const int64_t* seg_off, int32_t D, int64_t n_total,
                                         int32_t u_max, int32_t block_size, const int32_t* capacity,
                                         const int32_t* queue_len, const int32_t* a_prompt, const int32_t* a_upper,
                                         int64_t A, int32_t policy, int64_t rr_offset, int32_t* choice,
                                         int32_t* chosen_peak, int32_t* chosen_overflow, uint8_t* flags,
                                         int32_t* pair_peak, uint32_t* dev_err, hipStream_t stream) {
    if (D < 1 || n_total < 0 || A < 0 || rr_offset < 0 || u_max < 0 || u_max > MAPS_MAX_BLOCKS_U_MAX ||
        block_size < 1 || block_size > MAPS_MAX_BLOCK_SIZE || D > 65535)
        return MAPS_E_SIZE;
    if ((A + kTile - 1) / kTile > INT32_MAX) return MAPS_E_SIZE;
    if (policy != MAPS_POLICY_MQ && policy != MAPS_POLICY_MC) return MAPS_E_POLICY;
    if (!snapshot || !seg_off || !capacity || !queue_len || !dev_err ||
        (A > 0 && (!a_prompt || !a_upper || !choice || !chosen_peak || !chosen_overflow || !flags || !pair_peak)))
        return MAPS_E_NULL;
    if (A == 0) return MAPS_OK;
    const BlkLayout L = blk_layout(D, n_total, u_max, block_size);
    // chosen_overflow, chosen_peak and choice hold each tile's order, bounds and prompts until blocks_finish
    // writes them
    PairArgs pa{L, static_cast<const char*>(snapshot), a_prompt, a_upper, A, seg_off, pair_peak, chosen_overflow,
                chosen_peak, choice, dev_err};
    const int64_t tiles = (A + kTile - 1) / kTile;
    hipLaunchKernelGGL(blocks_order, dim3(unsigned(tiles)), dim3(kOrdNT), 0, stream, pa);
    MAPS_CHECK_LAUNCH();
    const int64_t rounds = (int64_t(D) + kXcds - 1) / kXcds;   // decoders per XCD
    if ((block_size & (block_size - 1)) == 0)
        hipLaunchKernelGGL(blocks_pairs<true>, dim3(unsigned(rounds * kXcds * tiles)), dim3(kPairsNT), 0, stream, pa,
                           tiles);
    else
        hipLaunchKernelGGL(blocks_pairs<false>, dim3(unsigned(rounds * kXcds * tiles)), dim3(kPairsNT), 0, stream, pa,
                           tiles);
    MAPS_CHECK_LAUNCH();
    FinArgs fa{dev_err, D, block_size, capacity, queue_len, a_upper, A, policy, rr_offset, pair_peak, choice, chosen_peak,
               chosen_overflow, flags};
    const int64_t fb = (A + kFinNT - 1) / kFinNT;
    hipLaunchKernelGGL(blocks_finish, dim3(unsigned(fb < 4096 ? fb : 4096)), dim3(kFinNT), 0, stream, fa);
    MAPS_CHECK_LAUNCH();
    return MAPS_OK;
}
