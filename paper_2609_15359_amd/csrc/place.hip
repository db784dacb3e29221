// Global placement (Sec. 3.3 and Algorithm 1, App. C) on gfx950.
//
// Every arrival is evaluated against every decoder's snapshot.  With the
// snapshot of maps_internal.hpp the projected peak of one pair is
//   e    = bits_before(word) + popcount(word & below(U))     (rank of U)
//   peak = max(p + max(PMX_e, S_e + U (N_e + 1), U), base)
// i.e. one 8-byte and one 16-byte LDS read and a handful of integer ops.
//
// Work decomposition: the decoders are split into G groups and the arrivals
// into tiles.  Workgroup b handles group b % G -- so with G dividing 8 all
// workgroups of a group run on the same XCDs and share their L2 -- and tile
// b / G.  Each thread keeps its arrivals in registers; the workgroup walks its
// decoders in order, stages each decoder's rank words and records in LDS, and
// evaluates all its arrivals against it, writing the decoder-major pair-peak
// row segment with coalesced stores and keeping the running best choice per
// arrival.  Ties keep the earlier (lower) decoder.  With G > 1 each group
// writes its best (key, decoder, peak) per arrival and place_reduce picks the
// best group in group order; with G = 1 the outputs are written directly.
//
// Selection key (smaller is better): policy MQ uses Q_d for a feasible pair
// and 2^31 | (peak - C_d) otherwise; policy MC uses (peak - C_d) + 2^31.
#include "maps_internal.hpp"

namespace maps {
namespace {

constexpr int kNT = 512;          // 8 waves per CU: 256 VGPRs per lane for the arrivals
constexpr size_t kLdsBytes = 160 * 1024;
constexpr int kMaxGroups = 8;

struct PlaceArgs {
    SnapLayout L;
    const void* snap;
    const int32_t* cap;
    const int32_t* qlen;
    const int32_t* ap;
    const int32_t* aU;
    int64_t A;
    int64_t rr_offset;
    int32_t* choice;
    int32_t* chosen_peak;
    int32_t* chosen_over;
    uint8_t* flags;
    int32_t* pair;
    uint32_t* pkey;   // [G][A] partial best keys
    int32_t* pdec;    // [G][A] partial best decoders
    int32_t* ppeak;   // [G][A] partial best peaks
    int32_t G;
    int32_t Dg;       // decoders per group
    int64_t rec_cap;  // records that fit LDS next to the rank words (0: rank words do not fit)
    uint32_t* dev_err;
};

__device__ inline bool snapshot_ok(const SnapHeader* h, const SnapLayout& L) {
    return h->magic == kSnapMagic && h->D == L.D && h->u_max == L.u_max && h->W == L.W;
}

__device__ inline int32_t imax(int32_t a, int32_t b) { return a > b ? a : b; }

// Per-thread state of kAPT arrivals: prompt, bound, bound clamped for the
// rank lookup, index of its rank word and the mask of the bits below it, and
// the best (key, decoder) seen so far.
template <int kAPT>
struct Arrivals {
    int32_t p[kAPT], U[kAPT], Ucl[kAPT];
    uint32_t wi[kAPT], mask[kAPT];
    uint32_t best_key[kAPT];
    int32_t best_d[kAPT];
};

// Projected peak of one arrival on one decoder, reading the snapshot in HBM.
__device__ __forceinline__ int32_t peak_from_hbm(const SnapView& V, int32_t W, int32_t d, int32_t p, int32_t U,
                                                 int32_t Ucl, uint32_t wi, uint32_t mask) {
    const DecHeader h = V.dec[d];
    const uint2 w = V.rank[int64_t(d) * W + wi];
    uint32_t e = w.y + __popc(w.x & mask);
    e = e < uint32_t(h.E) ? e : uint32_t(h.E);
    const int4 r = V.rec[h.rec_off + e];
    const int32_t lin = r.y + int32_t(__umul24(uint32_t(Ucl), uint32_t(r.z)));
    const int32_t pf = max(max(r.x, lin), U);
    return p + pf > h.base_peak ? p + pf : h.base_peak;
}

// Evaluate every arrival of the thread against one decoder whose rank words
// and records are at rank/rec (LDS or HBM), write the pair-peak row and keep
// the best choice.  `kFull`: every arrival of the tile exists.
// Selection key (smaller is better), with u = peak - C + 2^31:
//   MQ: u when infeasible (u > 2^31), else Q_d;   MC: u.
template <int kAPT, bool kFull, bool kPairs, int kPolicy>
__device__ __forceinline__ void eval_decoder(Arrivals<kAPT>& s, const uint2* rank, const int4* rec, int32_t E,
                                             int32_t base, int32_t C, int32_t Q, int32_t d, bool first,
                                             int32_t* prow, int64_t a0, int64_t A) {
    constexpr int kChunk = kAPT < 4 ? kAPT : 4;   // arrivals whose lookups are in flight together
    const uint32_t kC = 0x80000000u - uint32_t(C);
#pragma unroll
    for (int c = 0; c < kAPT; c += kChunk) {
        uint2 w[kChunk];
#pragma unroll
        for (int i = 0; i < kChunk; ++i) w[i] = rank[s.wi[c + i]];
        int4 r[kChunk];
#pragma unroll
        for (int i = 0; i < kChunk; ++i) {
            uint32_t e = w[i].y + __popc(w[i].x & s.mask[c + i]);
            e = e < uint32_t(E) ? e : uint32_t(E);   // stays inside the decoder's records
            r[i] = rec[e];
        }
#pragma unroll
        for (int i = 0; i < kChunk; ++i) {
            const int k = c + i;
            // PF(U) = max(PMX_e, S_e + U (N_e + 1)), U itself when beyond the last event
            const int32_t lin = r[i].y + int32_t(__umul24(uint32_t(s.Ucl[k]), uint32_t(r[i].z)));
            const int32_t pf = max(max(r[i].x, lin), s.U[k]);
            const int32_t peak = imax(s.p[k] + pf, base);
            if constexpr (kPairs) {
                // uniform row base per k, lane offset in a VGPR: no per-arrival 64-bit address
                int32_t* row = prow + a0 + int64_t(k) * kNT;
                if (kFull || a0 + int64_t(k) * kNT + threadIdx.x < A)
                    __builtin_nontemporal_store(s.U[k] < 0 ? -1 : peak, row + threadIdx.x);
            }
            const uint32_t u = uint32_t(peak) + kC;
            uint32_t key;
            if constexpr (kPolicy == MAPS_POLICY_MQ) key = u > 0x80000000u ? u : uint32_t(Q);
            else key = u;
            const bool take = first || key < s.best_key[k];
            s.best_key[k] = take ? key : s.best_key[k];
            s.best_d[k] = take ? d : s.best_d[k];
        }
    }
}

// A 16-byte unit as a native vector (kept in registers when staged).
typedef int32_t v4i __attribute__((ext_vector_type(4)));

// 16-byte unit u of decoder d's snapshot slice: its rank words, then its records.
__device__ __forceinline__ const int4* snapshot_unit(const SnapView& V, int32_t W, int32_t d, const DecHeader& h,
                                                     int64_t u) {
    const int64_t half_w = W / 2;
    return u < half_w ? reinterpret_cast<const int4*>(V.rank + int64_t(d) * W) + u : V.rec + h.rec_off + (u - half_w);
}

// Load this thread's first kPF units of decoder d into registers (units past
// the end re-read the last one, so every lane issues the same loads).
template <int kPF>
__device__ __forceinline__ void stage_units(v4i (&stage)[kPF], const SnapView& V, int32_t W, int32_t d,
                                            const DecHeader& h) {
    const int64_t last = int64_t(W / 2) + h.E;
#pragma unroll
    for (int j = 0; j < kPF; ++j) {
        const int64_t u = threadIdx.x + int64_t(j) * kNT;
        stage[j] = *reinterpret_cast<const v4i*>(snapshot_unit(V, W, d, h, u < last ? u : last));
    }
}

template <int kAPT, bool kFull, bool kPairs, bool kFinal, int kPolicy>
__device__ __forceinline__ void place_tile(const PlaceArgs& g, const SnapView& V, int4* lds, int32_t grp,
                                           int64_t a0) {
    constexpr int kPF = 7;   // 16-byte units per thread staged in registers ahead of use
    const SnapLayout& L = g.L;
    const int32_t W = L.W;
    const int32_t half_w = W / 2;              // rank words in 16-byte units
    const int32_t d_begin = grp * g.Dg;
    const int32_t d_end = d_begin + g.Dg < L.D ? d_begin + g.Dg : L.D;
    const int64_t max_tot = V.hdr->max_tot;
    const int64_t n_total = V.hdr->n_total;
    const int32_t ucl_max = 32 * W - 1;        // ranks above every event
    const int64_t lds_units = g.rec_cap > 0 ? half_w + g.rec_cap : 0;

    Arrivals<kAPT> s;
    bool neg = false, range = false;
#pragma unroll
    for (int k = 0; k < kAPT; ++k) {
        const int64_t a = a0 + int64_t(k) * kNT + threadIdx.x;
        int32_t p = 0, U = -1;
        if (kFull || a < g.A) { p = g.ap[a]; U = g.aU[a]; }
        neg |= p < 0;
        if (U >= 0 && int64_t(p) + U + max_tot + L.u_max > int64_t(INT32_MAX)) range = true;
        s.p[k] = p < 0 ? 0 : p;
        s.U[k] = U;
        const int32_t uc = U < 0 ? 0 : (U < ucl_max ? U : ucl_max);
        s.Ucl[k] = uc;
        s.wi[k] = uint32_t(uc >> 5);
        s.mask[k] = (1u << (uc & 31)) - 1u;
        s.best_key[k] = 0xFFFFFFFFu;
        s.best_d[k] = d_begin;
    }
    if (neg) raise_error(g.dev_err, MAPS_ERR_NEG_LEN);
    if (range) raise_error(g.dev_err, MAPS_ERR_INT32_RANGE);

    auto fits = [&](const DecHeader& h) { return h.E >= 0 && int64_t(half_w) + h.E + 1 <= lds_units; };
    auto ok = [&](const DecHeader& h) {
        return h.E >= 0 && h.rec_off >= 0 && h.rec_off + h.E + 1 <= n_total + L.D && h.base_peak >= 0;
    };

    v4i stage[kPF];
    DecHeader h = V.dec[d_begin < d_end ? d_begin : 0];
    if (d_begin < d_end && ok(h) && fits(h)) stage_units<kPF>(stage, V, W, d_begin, h);
    for (int32_t d = d_begin; d < d_end; ++d) {
        const int32_t C = g.cap[d], Q = g.qlen[d];
        if (threadIdx.x == 0 && (C < 0 || Q < 0)) raise_error(g.dev_err, MAPS_ERR_NEG_LEN);
        const bool valid = ok(h);
        const bool in_lds = valid && fits(h);
        if (!valid && threadIdx.x == 0) raise_error(g.dev_err, MAPS_ERR_SNAPSHOT);
        if (in_lds) {
            __syncthreads();   // every wave finished reading the previous decoder
            const int64_t units = int64_t(half_w) + h.E + 1;
#pragma unroll
            for (int j = 0; j < kPF; ++j) {   // lanes past the end write the spare unit
                const int64_t u = threadIdx.x + int64_t(j) * kNT;
                reinterpret_cast<v4i*>(lds)[u < units ? u : lds_units] = stage[j];
            }
            for (int64_t u = threadIdx.x + int64_t(kPF) * kNT; u < units; u += kNT) lds[u] = *snapshot_unit(V, W, d, h, u);
            __syncthreads();
        }
        const DecHeader cur = h;
        if (d + 1 < d_end) {
            h = V.dec[d + 1];
            if (ok(h) && fits(h)) stage_units<kPF>(stage, V, W, d + 1, h);   // overlaps the evaluation below
        }
        if (!valid) continue;
        int32_t* prow = kPairs ? g.pair + int64_t(d) * g.A : nullptr;
        if (in_lds)
            eval_decoder<kAPT, kFull, kPairs, kPolicy>(s, reinterpret_cast<const uint2*>(lds), lds + half_w, cur.E,
                                                        cur.base_peak, C, Q, d, d == d_begin, prow, a0, g.A);
        else
            eval_decoder<kAPT, kFull, kPairs, kPolicy>(s, V.rank + int64_t(d) * W, V.rec + cur.rec_off, cur.E,
                                                        cur.base_peak, C, Q, d, d == d_begin, prow, a0, g.A);
    }

#pragma unroll
    for (int k = 0; k < kAPT; ++k) {
        const int64_t a = a0 + int64_t(k) * kNT + threadIdx.x;
        if (!kFull && a >= g.A) continue;
        // the chosen pair's peak, evaluated once more from the snapshot in HBM
        const bool has = d_begin < d_end && s.U[k] >= 0 && ok(V.dec[s.best_d[k]]);
        const int32_t peak = has ? peak_from_hbm(V, W, s.best_d[k], s.p[k], s.U[k], s.Ucl[k], s.wi[k], s.mask[k]) : 0;
        if constexpr (kFinal) {
            if (s.U[k] < 0) {
                g.choice[a] = int32_t((g.rr_offset + a) % L.D);
                g.chosen_peak[a] = -1;
                g.chosen_over[a] = 0;
                g.flags[a] = 2;
            } else {
                const int32_t C = g.cap[s.best_d[k]];
                g.choice[a] = s.best_d[k];
                g.chosen_peak[a] = peak;
                g.chosen_over[a] = peak > C ? peak - C : 0;
                g.flags[a] = peak <= C ? 1 : 0;
            }
        } else {
            const int64_t o = int64_t(grp) * g.A + a;
            g.pkey[o] = d_begin < d_end ? s.best_key[k] : 0xFFFFFFFFu;
            g.pdec[o] = s.best_d[k] < L.D ? s.best_d[k] : 0;
            g.ppeak[o] = peak;
        }
    }
}

template <int kAPT, bool kPairs, bool kFinal, int kPolicy>
__global__ __launch_bounds__(kNT) void place_pairs(PlaceArgs g) {
    extern __shared__ int4 lds[];
    const SnapView V = snap_view(const_cast<void*>(g.snap), g.L);
    if (!snapshot_ok(V.hdr, g.L)) {
        if (blockIdx.x == 0 && threadIdx.x == 0) raise_error(g.dev_err, MAPS_ERR_SNAPSHOT);
        return;
    }
    const int32_t grp = blockIdx.x % g.G;
    const int64_t a0 = int64_t(blockIdx.x / g.G) * (kNT * kAPT);
    if (a0 + kNT * kAPT <= g.A)
        place_tile<kAPT, true, kPairs, kFinal, kPolicy>(g, V, lds, grp, a0);
    else
        place_tile<kAPT, false, kPairs, kFinal, kPolicy>(g, V, lds, grp, a0);
}

__global__ __launch_bounds__(256) void place_reduce(PlaceArgs g) {
    const SnapLayout& L = g.L;
    const SnapView V = snap_view(const_cast<void*>(g.snap), L);
    if (!snapshot_ok(V.hdr, L)) return;
    const int64_t stride = int64_t(gridDim.x) * blockDim.x;
    for (int64_t a = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; a < g.A; a += stride) {
        if (g.aU[a] < 0) {
            g.choice[a] = int32_t((g.rr_offset + a) % L.D);
            g.chosen_peak[a] = -1;
            g.chosen_over[a] = 0;
            g.flags[a] = 2;
            continue;
        }
        uint32_t key = g.pkey[a];
        int32_t d = g.pdec[a], peak = g.ppeak[a];
        for (int32_t gi = 1; gi < g.G; ++gi) {
            const int64_t o = int64_t(gi) * g.A + a;
            const uint32_t k2 = g.pkey[o];
            if (k2 < key) { key = k2; d = g.pdec[o]; peak = g.ppeak[o]; }
        }
        d = d < 0 || d >= L.D ? 0 : d;
        const int32_t C = g.cap[d];
        g.choice[a] = d;
        g.chosen_peak[a] = peak;
        g.chosen_over[a] = peak > C ? peak - C : 0;
        g.flags[a] = peak <= C ? 1 : 0;
    }
}

template <int kAPT, bool kPairs, bool kFinal, int kPolicy>
void launch_one(dim3 grid, size_t lds, hipStream_t s, const PlaceArgs& a) {
    auto fn = place_pairs<kAPT, kPairs, kFinal, kPolicy>;
    allow_dynamic_lds(fn, kLdsBytes);
    hipLaunchKernelGGL(fn, grid, dim3(kNT), lds, s, a);
}

template <int kAPT, bool kPairs, bool kFinal>
void launch_policy(int32_t policy, dim3 grid, size_t lds, hipStream_t s, const PlaceArgs& a) {
    if (policy == MAPS_POLICY_MQ) launch_one<kAPT, kPairs, kFinal, MAPS_POLICY_MQ>(grid, lds, s, a);
    else launch_one<kAPT, kPairs, kFinal, MAPS_POLICY_MC>(grid, lds, s, a);
}

template <int kAPT>
void launch_apt(bool pairs, bool final_, int32_t policy, dim3 grid, size_t lds, hipStream_t s, const PlaceArgs& a) {
    if (pairs) {
        if (final_) launch_policy<kAPT, true, true>(policy, grid, lds, s, a);
        else launch_policy<kAPT, true, false>(policy, grid, lds, s, a);
    } else {
        if (final_) launch_policy<kAPT, false, true>(policy, grid, lds, s, a);
        else launch_policy<kAPT, false, false>(policy, grid, lds, s, a);
    }
}

// Arrivals per thread and decoder groups: the largest arrival tile that still
// gives at least one workgroup per compute unit.
void plan(int32_t D, int64_t A, int cus, int* apt, int* groups) {
    for (int t : {8, 4, 2, 1}) {
        const int64_t tiles = (A + int64_t(kNT) * t - 1) / (int64_t(kNT) * t);
        int G = 1;
        while (G < kMaxGroups && G < D && tiles * G < cus) G *= 2;
        if (G > D) G = D;
        *apt = t;
        *groups = G;
        if (tiles * G >= cus) return;
    }
}

struct PlaceWorkspace {
    uint32_t* key;
    int32_t* dec;
    int32_t* peak;
    size_t bytes;
};

PlaceWorkspace place_carve(void* base, int64_t A) {
    PlaceWorkspace w;
    char* p = static_cast<char*>(base);
    size_t off = 0;
    auto take = [&](size_t bytes) { char* r = p ? p + off : nullptr; off += align256(bytes); return r; };
    w.key = reinterpret_cast<uint32_t*>(take(size_t(kMaxGroups) * A * 4));
    w.dec = reinterpret_cast<int32_t*>(take(size_t(kMaxGroups) * A * 4));
    w.peak = reinterpret_cast<int32_t*>(take(size_t(kMaxGroups) * A * 4));
    w.bytes = off;
    return w;
}

int compute_units() {
    int dev = 0, cus = 256;
    if (hipGetDevice(&dev) == hipSuccess) {
        int v = 0;
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && v > 0) cus = v;
    }
    return cus;
}

}  // namespace
}  // namespace maps

using namespace maps;

extern "C" size_t maps_place_workspace_size(int32_t D, int64_t A, int32_t u_max) {
    if (D < 1 || A < 0 || u_max < 0) return 0;
    return place_carve(nullptr, A).bytes;
}

extern "C" maps_status maps_place(const void* snapshot, int32_t D, int32_t u_max, const int32_t* capacity,
                                  const int32_t* queue_len, const int32_t* a_prompt, const int32_t* a_upper,
                                  int64_t A, int32_t policy, int64_t rr_offset, int32_t* choice,
                                  int32_t* chosen_peak, int32_t* chosen_overflow, uint8_t* flags,
                                  int32_t* pair_peak, uint32_t* dev_err, void* workspace,
                                  size_t workspace_bytes, hipStream_t stream) {
    if (D < 1 || A < 0 || rr_offset < 0 || u_max < 0 || u_max > MAPS_MAX_U_MAX) return MAPS_E_SIZE;
    if (policy != MAPS_POLICY_MQ && policy != MAPS_POLICY_MC) return MAPS_E_POLICY;
    if (!snapshot || !capacity || !queue_len || !dev_err ||
        (A > 0 && (!a_prompt || !a_upper || !choice || !chosen_peak || !chosen_overflow || !flags)))
        return MAPS_E_NULL;
    if (A == 0) return MAPS_OK;
    int apt = 8, G = 1;
    plan(D, A, compute_units(), &apt, &G);
    PlaceWorkspace w{};
    if (G > 1) {
        if (!workspace) return MAPS_E_NULL;
        w = place_carve(workspace, A);
        if (workspace_bytes < w.bytes) return MAPS_E_WORKSPACE;
    }
    PlaceArgs a;
    a.L = snap_layout(D, 0, u_max);
    a.snap = snapshot;
    a.cap = capacity;
    a.qlen = queue_len;
    a.ap = a_prompt;
    a.aU = a_upper;
    a.A = A;
    a.rr_offset = rr_offset;
    a.choice = choice;
    a.chosen_peak = chosen_peak;
    a.chosen_over = chosen_overflow;
    a.flags = flags;
    a.pair = pair_peak;
    a.pkey = w.key;
    a.pdec = w.dec;
    a.ppeak = w.peak;
    a.G = G;
    a.Dg = (D + G - 1) / G;
    a.dev_err = dev_err;
    // The record region starts after the rank words, whose offset does not
    // depend on the number of residents; records are addressed through the
    // decoder headers and bound-checked against the snapshot's own count.
    const size_t rank_bytes = size_t(a.L.W) * 8;
    // LDS: rank words, records, and one spare 16-byte unit
    a.rec_cap = rank_bytes + 64 * 16 <= kLdsBytes ? int64_t((kLdsBytes - rank_bytes) / 16) - 1 : 0;
    const size_t lds = a.rec_cap > 0 ? kLdsBytes : 0;
    const int64_t tiles = (A + int64_t(kNT) * apt - 1) / (int64_t(kNT) * apt);
    const dim3 grid(unsigned(tiles * G));
    const bool pairs = pair_peak != nullptr, final_ = G == 1;
    switch (apt) {
        case 8: launch_apt<8>(pairs, final_, policy, grid, lds, stream, a); break;
        case 4: launch_apt<4>(pairs, final_, policy, grid, lds, stream, a); break;
        case 2: launch_apt<2>(pairs, final_, policy, grid, lds, stream, a); break;
        default: launch_apt<1>(pairs, final_, policy, grid, lds, stream, a); break;
    }
    MAPS_CHECK_LAUNCH();
    if (!final_) {
        const int64_t blocks = (A + 255) / 256;
        hipLaunchKernelGGL(place_reduce, dim3(unsigned(blocks < 4096 ? blocks : 4096)), dim3(256), 0, stream, a);
        MAPS_CHECK_LAUNCH();
    }
    return MAPS_OK;
}
