// Global placement (Sec. 3.3 and Algorithm 1, App. C) on gfx950.
//
// Every arrival is evaluated against every decoder's snapshot.  With the
// snapshot of maps_internal.hpp the projected peak of one pair is either
//   e    = bits_before(word) + popcount(word & below(U))     (rank of U)
//   peak = max(p + max(PMX_e, S_e + U (N_e + 1), U), base)
// (record path: an 8-byte rank word and an 8-byte record, plus a second 8-byte
// record only past the event's threshold, all in LDS), or, when the snapshot
// carries dense profiles,
//   peak = max(p + max(F[min(U, u_max)], U), base)
// (profile path: one 4-byte LDS read).
//
// Work decomposition: the decoders are split into G groups and the arrivals
// into tiles.  Workgroup b handles group b % G -- so with G dividing 8 all
// workgroups of a group run on the same XCDs and share their L2 -- and tile
// b / G.  Each thread keeps its arrivals in registers; the workgroup walks its
// decoders in order, stages their snapshot data in LDS, and evaluates all its
// arrivals against each, writing the decoder-major pair-peak row segment with
// coalesced stores and keeping the running best choice per arrival (ties keep
// the earlier, lower decoder).  Each group writes its best (key, decoder) per
// arrival; place_finish picks the best group in group order, evaluates the
// chosen pair's peak once more from the snapshot and writes the outputs.
//
// Selection (smaller key is better, see select_key): policy MQ prefers any
// feasible decoder, by queue length, then the smallest overflow; policy MC
// the largest slack.
#include "maps_internal.hpp"
#include "order_core.hpp"

namespace maps {
namespace {

constexpr int kNT = 512;          // 8 waves per CU: 256 VGPRs per lane for the arrivals
constexpr size_t kLdsBytes = 160 * 1024;
constexpr size_t kRedBytes = 256;   // record path: the tile's bound reduction, past the two buffers
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
    int32_t* pkey;     // [G][A] best key of each group
    int32_t* pdec;     // [G][A] best decoder of each group (16-bit entries when dec16)
    int32_t G;
    int32_t policy;
    int32_t Dg;        // decoders per group
    int32_t buf_units; // record path: 16-byte units per LDS buffer (0: slices stay in HBM)
    int32_t nb;        // profile path: profiles per LDS batch
    uint32_t* dev_err;
    bool dec16;        // D <= 65,536: the groups' decoders are written as 16-bit indices
};

template <bool B>
struct BoolTag {
    static constexpr bool value = B;
};

// Read-only values every lane needs alike, loaded through the scalar cache.
template <typename T>
__device__ __forceinline__ T load_uniform(const T* p) {
    return *(const __attribute__((address_space(4))) T*)(p);
}

__device__ inline bool snapshot_ok(const SnapHeader* h, const SnapLayout& L) {
    return load_uniform(&h->magic) == kSnapMagic && load_uniform(&h->D) == L.D &&
           load_uniform(&h->u_max) == L.u_max && load_uniform(&h->W) == L.W && load_uniform(&h->P) == L.P;
}

__device__ inline int32_t imax(int32_t a, int32_t b) { return a > b ? a : b; }

// A 16-byte unit as a native vector (kept in registers when staged).
typedef int32_t v4i __attribute__((ext_vector_type(4)));

// Selection key of a pair as a signed value (smaller is better), with the
// overflow v = peak - C_d (|v| < 2^31):
//   MQ: v - 1 when infeasible (v > 0), else Q_d - 2^31 (every feasible pair
//       ranks first, by queue length);   MC: v (largest slack first).
// Qm is Q_d - 2^31.  The MQ key is a bit-select on the sign of v - 1 (no
// compare: a select on a fresh compare result costs wait states on gfx950).
template <int kPolicy>
__device__ __forceinline__ int32_t select_key(int32_t peak, int32_t C, int32_t Qm) {
    if constexpr (kPolicy == MAPS_POLICY_MQ) {
        const int32_t t = int32_t(uint32_t(peak) - uint32_t(C) - 1u);   // v - 1, exact: v > -2^31
        const int32_t m = t >> 31;                                       // all ones when feasible
        int32_t key;
        asm("v_bfi_b32 %0, %1, %2, %3" : "=v"(key) : "v"(m), "s"(Qm), "v"(t));   // m ? Qm : t
        return key;
    } else {
        return peak - C;
    }
}

// The peak behind a key that is not a feasible MQ key (MQ: key >= 0).
template <int kPolicy>
__device__ __forceinline__ int64_t key_peak(int32_t key, int32_t C) {
    return int64_t(key) + C + (kPolicy == MAPS_POLICY_MQ ? 1 : 0);
}

// Per-decoder values of up to 64 consecutive decoders, lane j of every wave
// holding decoder d0 + j.  One vector load per field serves 64 decoders, and
// each decoder's values are then read out of the lanes into scalar registers:
// no load latency per decoder, and no wait on a fresh load (which would also
// wait for every store issued before it) inside the decoder loop.
struct DecLanes {
    int32_t off_lo, off_hi, E, base, C, Q, pmx_end;
};

__device__ __forceinline__ DecLanes load_lanes(const PlaceArgs& g, const SnapView& V, int32_t d0, int32_t d_end) {
    const int32_t d = d0 + int32_t(threadIdx.x % kWave);
    DecLanes l{0, 0, -1, -1, 0, 0, 0};
    if (d < d_end) {
        const DecHeader h = V.dec[d];
        l.off_lo = int32_t(uint64_t(h.slice_off));
        l.off_hi = int32_t(uint64_t(h.slice_off) >> 32);
        l.E = h.E;
        l.base = h.base_peak;
        l.C = g.cap[d];
        l.Q = g.qlen[d];
        l.pmx_end = h.pmx_end;
    }
    return l;
}

__device__ __forceinline__ int32_t lane_value(int32_t v, int32_t lane) { return __builtin_amdgcn_readlane(v, lane); }

__device__ __forceinline__ DecHeader lane_header(const DecLanes& l, int32_t lane) {
    DecHeader h;
    h.slice_off = int64_t(uint64_t(uint32_t(lane_value(l.off_lo, lane))) |
                          (uint64_t(uint32_t(lane_value(l.off_hi, lane))) << 32));
    h.tot = 0;
    h.E = lane_value(l.E, lane);
    h.base_peak = lane_value(l.base, lane);
    h.hot_lo = 1;
    h.hot_hi = 0;
    h.flat_lo = 1;
    h.pmx_end = lane_value(l.pmx_end, lane);
    for (int i = 0; i < 6; ++i) h.pad[i] = 0;
    return h;
}

// Largest total demand sum_r (p + g + R) and record count E + 1 over the
// decoders [d0, d1), and the intersection of their hot windows, the same in
// every lane.
struct GroupMax {
    int64_t tot;
    int32_t records;
    int32_t hot_lo, hot_hi;
    int32_t flat_lo;   // largest max(flat_lo, hot_lo)
};

__device__ inline GroupMax group_max(const SnapView& V, int32_t d0, int32_t d1) {
    int64_t t = 0;
    int32_t r = 0, lo = 0, hi = INT32_MAX, fl = 0;
    for (int32_t d = d0 + int32_t(threadIdx.x % kWave); d < d1; d += kWave) {
        const DecHeader h = V.dec[d];
        t = t > h.tot ? t : h.tot;
        r = r > h.E + 1 ? r : h.E + 1;
        lo = lo > h.hot_lo ? lo : h.hot_lo;
        hi = hi < h.hot_hi ? hi : h.hot_hi;
        fl = fl > h.flat_lo ? fl : h.flat_lo;
    }
    lo = wave_reduce_max(lo);
    fl = wave_reduce_max(fl);
    return GroupMax{wave_reduce_max(t), wave_reduce_max(r), lo, -wave_reduce_max(-hi), fl > lo ? fl : lo};
}

// Raw buffer resources (gfx9 descriptor, 32-bit data format): accesses whose
// VGPR offset (plus immediate) reaches past `bytes` read 0 and write nothing.
constexpr int kBufferWord3 = 0x00020000;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, int(bytes), kBufferWord3);
}

// Pair-peak store of arrival k of the thread into a tile row.  In a full tile
// the arrival's place in the row is a uniform offset; in a partial tile the
// whole offset goes through the range check, which drops the missing arrivals.
// Plain write-back stores: the non-temporal hint made the pass 12% slower.
template <bool kFull>
__device__ __forceinline__ void store_pair(__amdgpu_buffer_rsrc_t row, int k, int32_t v) {
    if constexpr (kFull)
        __builtin_amdgcn_raw_buffer_store_b32(v, row, int(threadIdx.x) * 4, k * kNT * 4, 0);
    else
        __builtin_amdgcn_raw_buffer_store_b32(v, row, int(threadIdx.x) * 4 + k * kNT * 4, 0, 0);
}

// Projected peak of (p, U) from the records of event e (see maps_internal.hpp):
// PF(U) = PMX_e below the event's threshold, else S_e + U (N_e + 1).  For a
// bound at or above 32 W the rank lands on event E (N + 1 = 1, S = 0), where
// S + U (N + 1) = U; so the product may use U itself (its low 24 bits, all of
// it whenever an event before E is hit, since events are <= u_max), and the
// final max with U restores it.
__device__ __forceinline__ int32_t event_peak(const int32_t* pmx, const int32_t* thr, const int2* cold, uint32_t e,
                                              int32_t p, int32_t U, int32_t base) {
    int32_t pf = max(pmx[e], U);
    if (U >= thr[e]) {
        const int2 c = cold[e];
        pf = max(c.x + int32_t(__umul24(uint32_t(U), uint32_t(c.y))), U);
    }
    return imax(p + pf, base);
}

// Raw prompt and bound of arrival k of the thread's tile (bound -1 past the
// batch).  Issued first in a workgroup: nothing else is needed to address
// them, so their latency overlaps the snapshot's header reads.
template <int kAPT>
__device__ __forceinline__ void fetch_arrivals(const PlaceArgs& g, int64_t a0, int32_t (&p)[kAPT],
                                               int32_t (&U)[kAPT]) {
#pragma unroll
    for (int k = 0; k < kAPT; ++k) {
        const int64_t a = a0 + int64_t(k) * kNT + threadIdx.x;
        p[k] = 0;
        U[k] = -1;
        if (a < g.A) { p[k] = g.ap[a]; U[k] = g.aU[a]; }
    }
}

// The fetched arrivals with their prompts clamped at 0, reporting the error
// bits of the tile's arrivals.
template <int kAPT>
__device__ __forceinline__ void check_arrivals(const PlaceArgs& g, int64_t max_tot, const int32_t (&rp)[kAPT],
                                               const int32_t (&rU)[kAPT], int32_t (&p)[kAPT], int32_t (&U)[kAPT]) {
    bool neg = false, range = false;
#pragma unroll
    for (int k = 0; k < kAPT; ++k) {
        const int32_t pk = rp[k], Uk = rU[k];
        neg |= pk < 0;
        if (Uk >= 0 && int64_t(pk) + Uk + max_tot + g.L.u_max > int64_t(INT32_MAX)) range = true;
        p[k] = pk < 0 ? 0 : pk;
        U[k] = Uk;
    }
    if (neg) raise_error(g.dev_err, MAPS_ERR_NEG_LEN);
    if (range) raise_error(g.dev_err, MAPS_ERR_INT32_RANGE);
}

// The group's best (key, decoder) of each arrival of the tile.
template <int kAPT, bool kFull>
__device__ __forceinline__ void write_partials(const PlaceArgs& g, int32_t grp, int64_t a0,
                                               const int32_t (&key)[kAPT], const int32_t (&dec)[kAPT]) {
#pragma unroll
    for (int k = 0; k < kAPT; ++k) {
        const int64_t a = a0 + int64_t(k) * kNT + threadIdx.x;
        if (!kFull && a >= g.A) continue;
        const int64_t o = int64_t(grp) * g.A + a;
        const int32_t d = dec[k] < g.L.D ? dec[k] : 0;
        g.pkey[o] = key[k];
        if (g.dec16) reinterpret_cast<uint16_t*>(g.pdec)[o] = uint16_t(d);
        else g.pdec[o] = d;
    }
}

// ---------------------------------------------------------------------------
// Record path.
//
// Each thread holds kAPT arrivals: prompt, bound, -1/0 for a missing bound,
// the LDS address of the bound's rank word in buffer 0 and the mask of the
// bits below it (bound clamped to [0, 32 W - 1]), and the running best.
// The workgroup walks its decoders with two LDS buffers: while decoder d is
// evaluated from one buffer, the rank words and PMX values of decoder d+1
// (and its cold records {S_e, N_e + 1}, unless the tile lies in every
// decoder's hot window) are already on their way into registers, and they
// are written to the other buffer before the single barrier of the next
// step.  Every lookup then stays in LDS.  A slice whose staged part exceeds
// a buffer is read from HBM altogether (with the thresholds, so that only
// lanes past one read a cold record).
// ---------------------------------------------------------------------------
constexpr int kStage = 7;   // 16-byte units per thread staged in registers: a whole LDS buffer

template <int kAPT>
struct RecArrivals {
    int32_t p[kAPT], U[kAPT], neg[kAPT];
    int32_t pU[kAPT];   // p + U, set by the walk without threshold tests
    uint32_t roff[kAPT], mask[kAPT];
    int32_t best_key[kAPT], best_d[kAPT];
};

// Evaluate the thread's arrivals against one decoder whose PMX values are at
// `pmx` and thresholds at `thr`, with its cold records at `cold` in HBM.  The
// thread's rank-word offsets are LDS addresses of buffer 0: with kLds the rank
// words are read at those addresses plus `rank_lds` (the buffer's offset, a
// constant where the buffer is fixed), otherwise at `rank_g` plus them (the
// HBM rank words minus buffer 0's LDS address).  Only lanes whose bound reaches an event's
// threshold read its cold record.  kHot: every bound of the tile lies in the
// decoder's hot window (no threshold test) and every arrival has a bound.
template <int kAPT, bool kFull, bool kPairs, int kPolicy, bool kHot, bool kLds>
__device__ __forceinline__ void eval_records(RecArrivals<kAPT>& s, const char* rank_g, uint32_t rank_lds,
                                             const int32_t* pmx, const int32_t* thr, const int2* cold, uint32_t E,
                                             int32_t base, int32_t C, int32_t Q, int32_t d,
                                             __amdgpu_buffer_rsrc_t row) {
    constexpr int kChunk = kAPT < 4 ? kAPT : 4;   // arrivals whose lookups are in flight together
    int32_t Qm = int32_t(uint32_t(Q) + 0x80000000u);
    asm("" : "+s"(Qm));   // kept as is in a scalar register: the key select then needs no source modifier
#pragma unroll
    for (int c = 0; c < kAPT; c += kChunk) {
        uint2 w[kChunk];
#pragma unroll
        for (int i = 0; i < kChunk; ++i) {
            if constexpr (kLds) {
                const uint64_t x =
                    *reinterpret_cast<const __attribute__((address_space(3))) uint64_t*>(size_t(s.roff[c + i] + rank_lds));
                w[i] = make_uint2(uint32_t(x), uint32_t(x >> 32));
            } else
                w[i] = *reinterpret_cast<const uint2*>(rank_g + s.roff[c + i]);
        }
        uint32_t e[kChunk];
        int32_t m[kChunk], t[kChunk];
#pragma unroll
        for (int i = 0; i < kChunk; ++i) {
            e[i] = w[i].y + __popc(w[i].x & s.mask[c + i]);
            if constexpr (kHot)   // LDS only: a rank past E (malformed slice) reads other LDS data, or 0
                asm("" : "+v"(e[i]));   // opaque: the table address stays one shift-add
            else
                e[i] = e[i] < E ? e[i] : E;   // stays inside the decoder's records
            m[i] = pmx[e[i]];
            if constexpr (!kHot) t[i] = thr[e[i]];
        }
        int32_t pf[kChunk];
        bool line = false;
#pragma unroll
        for (int i = 0; i < kChunk; ++i) {
            pf[i] = max(m[i], s.U[c + i]);
            if constexpr (!kHot) line |= s.U[c + i] >= t[i];
        }
        if (!kHot && __builtin_amdgcn_ballot_w64(line) != 0) {   // a lane of the wave reached a threshold
#pragma unroll
            for (int i = 0; i < kChunk; ++i) {
                const int32_t U = s.U[c + i];
                if (U >= t[i]) {
                    const int2 cr = cold[e[i]];
                    pf[i] = max(cr.x + int32_t(__umul24(uint32_t(U), uint32_t(cr.y))), U);
                }
            }
        }
#pragma unroll
        for (int i = 0; i < kChunk; ++i) {
            const int k = c + i;
            // without a threshold test pf = max(PMX, U), and p + pf = max(p + PMX, p + U)
            const int32_t peak = kHot ? imax(imax(s.p[k] + m[i], s.pU[k]), base) : imax(s.p[k] + pf[i], base);
            if constexpr (kPairs) store_pair<kFull>(row, k, kHot ? peak : peak | s.neg[k]);
            const int32_t key = select_key<kPolicy>(peak, C, Qm);
            const bool take = key < s.best_key[k];
            s.best_key[k] = take ? key : s.best_key[k];
            s.best_d[k] = take ? d : s.best_d[k];
        }
    }
}

// Evaluate the thread's arrivals against one decoder whose bounds all lie in
// its flat region (and hot window): PF(U) = max(PMX_E, U), so the peak is
// max(p + PMX_E, p + U, base) with no lookup.
template <int kAPT, bool kFull, bool kPairs, int kPolicy>
__device__ __forceinline__ void eval_flat(RecArrivals<kAPT>& s, int32_t pmx_end, int32_t base, int32_t C, int32_t Q,
                                          int32_t d, __amdgpu_buffer_rsrc_t row) {
    int32_t Qm = int32_t(uint32_t(Q) + 0x80000000u);
    asm("" : "+s"(Qm));
#pragma unroll
    for (int k = 0; k < kAPT; ++k) {
        const int32_t peak = imax(imax(s.p[k] + pmx_end, s.pU[k]), base);
        if constexpr (kPairs) store_pair<kFull>(row, k, peak);
        const int32_t key = select_key<kPolicy>(peak, C, Qm);
        const bool take = key < s.best_key[k];
        s.best_key[k] = take ? key : s.best_key[k];
        s.best_d[k] = take ? d : s.best_d[k];
    }
}

// Load this thread's units of `units` staged units of a slice into
// registers: rows j of kNT units that hold part of them (a uniform test).
// Staged unit u comes from slice unit u below `split` and from u + skip at
// or above it (the cold records follow the PMX values once the thresholds
// are skipped); units past the slice's end read as 0.
__device__ __forceinline__ void stage_slice(v4i (&stage)[kStage], const int4* src, int32_t units, int32_t split,
                                            int32_t skip) {
    const __amdgpu_buffer_rsrc_t rs = buffer_rsrc(src, uint32_t(units + skip) * 16u);
#pragma unroll
    for (int j = 0; j < kStage; ++j)
        if (j * kNT < units) {
            const int32_t u = int32_t(threadIdx.x) + j * kNT;
            stage[j] = __builtin_bit_cast(
                v4i, __builtin_amdgcn_raw_buffer_load_b128(rs, (u + (u >= split ? skip : 0)) * 16, 0, 0));
        }
}

// Evaluate the thread's arrivals against one decoder whose rank words, PMX
// values and cold records are all in LDS: PF(U) = max(PMX_e, S_e + U (N_e +
// 1), U) for every lane, with no threshold test (see event_peak for why the
// low 24 bits of U suffice in the product).
template <int kAPT, bool kFull, bool kPairs, int kPolicy>
__device__ __forceinline__ void eval_cold(RecArrivals<kAPT>& s, uint32_t rank_lds, const int32_t* pmx,
                                          const int2* cold, uint32_t E, int32_t base, int32_t C, int32_t Q,
                                          int32_t d, __amdgpu_buffer_rsrc_t row) {
    constexpr int kChunk = kAPT < 4 ? kAPT : 4;
    int32_t Qm = int32_t(uint32_t(Q) + 0x80000000u);
    asm("" : "+s"(Qm));
#pragma unroll
    for (int c = 0; c < kAPT; c += kChunk) {
        uint32_t e[kChunk];
#pragma unroll
        for (int i = 0; i < kChunk; ++i) {
            const uint64_t x =
                *reinterpret_cast<const __attribute__((address_space(3))) uint64_t*>(size_t(s.roff[c + i] + rank_lds));
            e[i] = uint32_t(x >> 32) + __popc(uint32_t(x) & s.mask[c + i]);
            e[i] = e[i] < E ? e[i] : E;   // stays inside the decoder's records
        }
        int32_t m[kChunk];
        int2 cr[kChunk];
#pragma unroll
        for (int i = 0; i < kChunk; ++i) {
            m[i] = pmx[e[i]];
            cr[i] = cold[e[i]];
        }
#pragma unroll
        for (int i = 0; i < kChunk; ++i) {
            const int k = c + i;
            const int32_t U = s.U[k];
            const int32_t lin = cr[i].x + int32_t(__umul24(uint32_t(U), uint32_t(cr[i].y)));
            const int32_t pf = imax(imax(m[i], lin), U);
            const int32_t peak = imax(s.p[k] + pf, base);
            if constexpr (kPairs) store_pair<kFull>(row, k, peak | s.neg[k]);
            const int32_t key = select_key<kPolicy>(peak, C, Qm);
            const bool take = key < s.best_key[k];
            s.best_key[k] = take ? key : s.best_key[k];
            s.best_d[k] = take ? d : s.best_d[k];
        }
    }
}

// 16-byte units of a decoder's cold records {S_e, N_e + 1}, e = 0..E.
__device__ __forceinline__ int64_t cold_units(int64_t E) { return (E + 2) / 2; }

// One arrival tile against the decoders of group grp.  kMixed: some slices
// may exceed an LDS buffer and are then read from HBM; otherwise every slice
// fits (a header claiming more is reported and skipped).
template <int kAPT, bool kFull, bool kPairs, int kPolicy, bool kMixed>
__device__ __forceinline__ void records_tile(const PlaceArgs& g, const SnapView& V, int4* lds, int32_t grp,
                                             int64_t a0, const GroupMax& gm, const int32_t (&rp)[kAPT],
                                             const int32_t (&rU)[kAPT], const DecLanes& first_lanes) {
    const SnapLayout& L = g.L;
    const int32_t half_w = L.W / 2;                // rank words in 16-byte units
    const int32_t d_begin = grp * g.Dg;
    const int32_t d_end = d_begin + g.Dg < L.D ? d_begin + g.Dg : L.D;
    const int64_t n_total = load_uniform(&V.hdr->n_total);
    const int32_t ucl_max = 32 * L.W - 1;          // ranks above every event
    const int32_t buf_units = g.buf_units;
    const int64_t tile_n = g.A - a0 < kNT * kAPT ? g.A - a0 : kNT * kAPT;

    // LDS address of buffer 0 (where the dynamic LDS starts)
    const uint32_t lds_off = uint32_t(size_t((__attribute__((address_space(3))) char*)lds));
    RecArrivals<kAPT> s;
    check_arrivals<kAPT>(g, gm.tot, rp, rU, s.p, s.U);
#pragma unroll
    for (int k = 0; k < kAPT; ++k) {
        const int32_t U = s.U[k];
        s.neg[k] = U < 0 ? -1 : 0;
        const int32_t uc = U < 0 ? 0 : (U < ucl_max ? U : ucl_max);
        s.roff[k] = uint32_t(uc >> 5) * 8u + lds_off;
        asm("" : "+v"(s.roff[k]));   // opaque: kept whole, so a read adds only an immediate offset
        s.mask[k] = (1u << (uc & 31)) - 1u;
        s.best_key[k] = INT32_MAX;
        s.best_d[k] = d_begin;
    }
    // smallest and largest bound of the tile, and whether an arrival lacks one
    // (reduced through LDS past the two buffers: with no static LDS the
    // buffers start at address 0, so their offsets fold into the LDS reads)
    int32_t (*red)[kNT / kWave] = reinterpret_cast<int32_t (*)[kNT / kWave]>(lds + 2 * buf_units);
    int32_t t_lo = INT32_MAX, t_hi = -1, t_neg = 0;
#pragma unroll
    for (int k = 0; k < kAPT; ++k) {
        const int32_t U = s.U[k];
        if (U >= 0) {
            t_lo = U < t_lo ? U : t_lo;
            t_hi = U > t_hi ? U : t_hi;
        } else if (int64_t(k) * kNT + threadIdx.x < tile_n) {
            t_neg = 1;
        }
    }
    t_lo = -wave_reduce_max(-t_lo);
    t_hi = wave_reduce_max(t_hi);
    t_neg = wave_reduce_max(t_neg);
    if (threadIdx.x % kWave == 0) {
        red[0][threadIdx.x / kWave] = t_lo;
        red[1][threadIdx.x / kWave] = t_hi;
        red[2][threadIdx.x / kWave] = t_neg;
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kNT / kWave; ++i) {
        t_lo = red[0][i] < t_lo ? red[0][i] : t_lo;
        t_hi = red[1][i] > t_hi ? red[1][i] : t_hi;
        t_neg |= red[2][i];
    }
    t_lo = __builtin_amdgcn_readfirstlane(t_lo);   // the same in every lane: keep the test below scalar
    t_hi = __builtin_amdgcn_readfirstlane(t_hi);
    t_neg = __builtin_amdgcn_readfirstlane(t_neg);
    // the tile skips every threshold test when the hot windows of all the
    // group's decoders hold all its bounds (and every arrival has a bound)
    const bool all_hot = !kMixed && t_neg == 0 && t_lo >= gm.hot_lo && t_hi <= gm.hot_hi;
    // ... and needs no lookup at all when they also lie in every flat region
    const bool all_flat = t_neg == 0 && t_lo >= gm.flat_lo && t_hi <= gm.hot_hi;

    // the decoder walk, with or without the threshold tests: it stages the
    // rank words and the PMX values, and the thresholds when it tests them
    auto walk = [&](auto hot_tag) {
        constexpr bool kHot = decltype(hot_tag)::value;
        if constexpr (kHot) {
#pragma unroll
            for (int k = 0; k < kAPT; ++k) {
                s.pU[k] = s.p[k] + s.U[k];
                asm("" : "+v"(s.pU[k]));   // opaque: keeps max(p + PMX, p + U, base) a single three-way max
            }
        }
        // staged units: rank words and PMX, and (full walk) the cold records after them
        auto staged = [&](const DecHeader& h) {
            return int64_t(half_w) + event_units(h.E) + (kHot ? 0 : cold_units(h.E));
        };
        auto fits = [&](const DecHeader& h) { return staged(h) <= buf_units; };
        auto stage_next = [&](v4i (&st)[kStage], const DecHeader& h) {
            const int32_t split = half_w + int32_t(event_units(h.E));
            stage_slice(st, V.slices + h.slice_off, int32_t(staged(h)), split,
                        kHot ? 0 : int32_t(event_units(h.E)));   // the cold records skip the thresholds
        };
        // loaded here rather than with the tile's first loads: holding them
        // across the preamble costs this walk registers and time
        DecLanes lanes = load_lanes(g, V, d_begin, d_end);
        int32_t lanes0 = d_begin;
        v4i stage[kStage];
        DecHeader h = lane_header(lanes, 0);
        bool h_ok = d_begin < d_end && slice_ok(h, n_total, L) && (kMixed || fits(h));
        if (h_ok && fits(h)) stage_next(stage, h);
        // one step per decoder; unrolled by two so that the buffer is a
        // compile-time offset where every slice is staged in LDS
        auto step = [&](int32_t d, auto par_tag) {
            constexpr bool kOdd = decltype(par_tag)::value;
            const DecHeader cur = h;
            const bool valid = h_ok;
            const bool in_lds = valid && (!kMixed || fits(cur));
            const int32_t C = lane_value(lanes.C, d - lanes0), Q = lane_value(lanes.Q, d - lanes0);
            if (threadIdx.x == 0 && (C < 0 || Q < 0)) raise_error(g.dev_err, MAPS_ERR_NEG_LEN);
            if (!valid && threadIdx.x == 0) raise_error(g.dev_err, MAPS_ERR_SNAPSHOT);
            int4* slice = lds + (kOdd ? (kMixed ? buf_units : kStage * kNT) : 0);
            if (in_lds) {
                // This buffer was last read for decoder d-2, which every wave
                // finished before passing the barrier of decoder d-1.  Staged
                // units past the slice's end (0) stay inside the buffer:
                // kStage * kNT units fit it.
                const int32_t units = int32_t(staged(cur));
#pragma unroll
                for (int j = 0; j < kStage; ++j)
                    if (j * kNT < units) reinterpret_cast<v4i*>(slice)[int(threadIdx.x) + j * kNT] = stage[j];
            }
            if (d + 1 < d_end) {
                if (d + 1 - lanes0 == kWave) {
                    lanes = load_lanes(g, V, d + 1, d_end);
                    lanes0 = d + 1;
                }
                h = lane_header(lanes, d + 1 - lanes0);
                h_ok = slice_ok(h, n_total, L) && (kMixed || fits(h));
                if (h_ok && fits(h))   // overlaps the evaluation
                    stage_next(stage, h);
            }
            __syncthreads();
            if (!valid) return;
            const __amdgpu_buffer_rsrc_t row =
                buffer_rsrc(kPairs ? g.pair + int64_t(d) * g.A + a0 : nullptr, kPairs ? uint32_t(tile_n) * 4u : 0u);
            if (!kMixed || in_lds) {
                const int32_t* pmx = reinterpret_cast<const int32_t*>(slice + half_w);
                const uint32_t rank_lds = kOdd ? uint32_t(kMixed ? buf_units : kStage * kNT) * 16u : 0u;
                if constexpr (kHot)
                    eval_records<kAPT, kFull, kPairs, kPolicy, true, true>(
                        s, nullptr, rank_lds, pmx, nullptr, nullptr, uint32_t(cur.E), cur.base_peak, C, Q, d, row);
                else
                    eval_cold<kAPT, kFull, kPairs, kPolicy>(
                        s, rank_lds, pmx, reinterpret_cast<const int2*>(slice + half_w + event_units(cur.E)),
                        uint32_t(cur.E), cur.base_peak, C, Q, d, row);
            } else if constexpr (kMixed) {
                eval_records<kAPT, kFull, kPairs, kPolicy, false, false>(
                    s, reinterpret_cast<const char*>(slice_rank(V, cur)) - lds_off, 0u, slice_pmx(V, cur, L),
                    slice_thr(V, cur, L), slice_cold(V, cur, L), uint32_t(cur.E), cur.base_peak, C, Q, d, row);
            }
        };
        for (int32_t d = d_begin; d < d_end; d += 2) {
            step(d, BoolTag<false>{});
            if (d + 1 < d_end) step(d + 1, BoolTag<true>{});
        }
    };
    // the walk of a tile in every flat region: no slices, no LDS, no barrier
    auto flat_walk = [&]() {
#pragma unroll
        for (int k = 0; k < kAPT; ++k) {
            s.pU[k] = s.p[k] + s.U[k];
            asm("" : "+v"(s.pU[k]));   // opaque: keeps max(p + PMX_E, p + U, base) a single three-way max
        }
        DecLanes lanes = first_lanes;
        int32_t lanes0 = d_begin;
        for (int32_t d = d_begin; d < d_end; ++d) {
            if (d - lanes0 == kWave) {
                lanes = load_lanes(g, V, d, d_end);
                lanes0 = d;
            }
            const DecHeader h = lane_header(lanes, d - lanes0);
            const int32_t C = lane_value(lanes.C, d - lanes0), Q = lane_value(lanes.Q, d - lanes0);
            const bool valid = slice_ok(h, n_total, L);
            if (threadIdx.x == 0 && (C < 0 || Q < 0)) raise_error(g.dev_err, MAPS_ERR_NEG_LEN);
            if (!valid && threadIdx.x == 0) raise_error(g.dev_err, MAPS_ERR_SNAPSHOT);
            if (!valid) continue;
            const __amdgpu_buffer_rsrc_t row =
                buffer_rsrc(kPairs ? g.pair + int64_t(d) * g.A + a0 : nullptr, kPairs ? uint32_t(tile_n) * 4u : 0u);
            eval_flat<kAPT, kFull, kPairs, kPolicy>(s, h.pmx_end, h.base_peak, C, Q, d, row);
        }
    };
    if (all_flat) flat_walk();
    else if (all_hot) walk(BoolTag<true>{});
    else walk(BoolTag<false>{});
    write_partials<kAPT, kFull>(g, grp, a0, s.best_key, s.best_d);
}

// When every slice of the group fits an LDS buffer the tile runs in one pass;
// otherwise it is split into sub-tiles of at most 4 arrivals per thread that
// read the large slices from HBM.
template <int kAPT, bool kPairs, int kPolicy>
__global__ __launch_bounds__(kNT) void place_records(PlaceArgs g) {
    extern __shared__ int4 lds[];
    const SnapView V = snap_view(const_cast<void*>(g.snap), g.L);
    const int32_t grp = blockIdx.x % g.G;
    const int64_t a0 = int64_t(blockIdx.x / g.G) * (kNT * kAPT);
    const int32_t d_begin = grp * g.Dg;
    const int32_t d_end = d_begin + g.Dg < g.L.D ? d_begin + g.Dg : g.L.D;
    // The tile's arrivals go out first (they need nothing but the arguments),
    // so their latency overlaps the snapshot header's check; the decoder
    // headers are read only once the header shows that the buffer holds them,
    // the first 64 decoders' values (for the flat walk) and the group's
    // maxima together.
    int32_t rp[kAPT], rU[kAPT];
    fetch_arrivals<kAPT>(g, a0, rp, rU);
    if (!snapshot_ok(V.hdr, g.L)) {
        if (blockIdx.x == 0 && threadIdx.x == 0) raise_error(g.dev_err, MAPS_ERR_SNAPSHOT);
        return;
    }
    const DecLanes lanes = load_lanes(g, V, d_begin, d_end);
    const GroupMax gm = group_max(V, d_begin, d_end);
    // the full walk stages rank words, PMX values and cold records: (E + 1) records of 4 + 8 bytes
    if (g.L.W / 2 + (int64_t(gm.records) + 3) / 4 + (int64_t(gm.records) + 1) / 2 <= g.buf_units) {
        if (a0 + kNT * kAPT <= g.A)
            records_tile<kAPT, true, kPairs, kPolicy, false>(g, V, lds, grp, a0, gm, rp, rU, lanes);
        else
            records_tile<kAPT, false, kPairs, kPolicy, false>(g, V, lds, grp, a0, gm, rp, rU, lanes);
    } else {
        constexpr int kSub = kAPT < 4 ? kAPT : 4;
        for (int t = 0; t < kAPT / kSub; ++t) {
            const int64_t b0 = a0 + int64_t(t) * kNT * kSub;
            if (b0 >= g.A) continue;
            int32_t sp[kSub], sU[kSub];
            fetch_arrivals<kSub>(g, b0, sp, sU);
            records_tile<kSub, false, kPairs, kPolicy, true>(g, V, lds, grp, b0, gm, sp, sU, lanes);
        }
    }
}

// ---------------------------------------------------------------------------
// Profile path (snapshots with P > 0).
//
// The profile F of a decoder answers a pair with one 4-byte LDS read:
//   peak = max(p + max(F[min(U, u_max)], U), base).
// The group's profiles go through LDS nb decoders at a time; while one batch
// is evaluated the next one is already on its way into registers.
// ---------------------------------------------------------------------------
constexpr int kProfPF = 16;

template <int kAPT>
struct ProfArrivals {
    int32_t p[kAPT], U[kAPT], neg[kAPT];
    uint32_t off[kAPT];   // byte offset of F[min(U, u_max)] in a profile
    int32_t best_key[kAPT], best_d[kAPT];
};

// Load this thread's units of the batch starting at decoder db (rows j of kNT
// units that hold part of it; units past its end read as 0).
__device__ __forceinline__ void stage_profile(v4i (&stage)[kProfPF], const int32_t* prof, int32_t P, int32_t db,
                                              int32_t units) {
    const __amdgpu_buffer_rsrc_t rs = buffer_rsrc(prof + int64_t(db) * P, uint32_t(units) * 16u);
#pragma unroll
    for (int j = 0; j < kProfPF; ++j)
        if (j * kNT < units)
            stage[j] = __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(
                                                   rs, int(threadIdx.x) * 16 + j * kNT * 16, 0, 0));
}

template <int kAPT, bool kFull, bool kPairs, int kPolicy>
__device__ __forceinline__ void prof_decoder(ProfArrivals<kAPT>& s, const char* table, int32_t base, int32_t C,
                                             int32_t Q, int32_t d, __amdgpu_buffer_rsrc_t row) {
    const int32_t Qm = int32_t(uint32_t(Q) + 0x80000000u);
#pragma unroll
    for (int k = 0; k < kAPT; ++k) {
        const int32_t f = *reinterpret_cast<const int32_t*>(table + s.off[k]);
        const int32_t peak = imax(s.p[k] + (f > s.U[k] ? f : s.U[k]), base);
        if constexpr (kPairs) store_pair<kFull>(row, k, peak | s.neg[k]);
        const int32_t key = select_key<kPolicy>(peak, C, Qm);
        const bool take = key < s.best_key[k];
        s.best_key[k] = take ? key : s.best_key[k];
        s.best_d[k] = take ? d : s.best_d[k];
    }
}

template <int kAPT, bool kFull, bool kPairs, int kPolicy>
__device__ __forceinline__ void prof_tile(const PlaceArgs& g, const SnapView& V, int4* lds, int32_t grp,
                                          int64_t a0) {
    const SnapLayout& L = g.L;
    const int32_t P = L.P;
    const int32_t d_begin = grp * g.Dg;
    const int32_t d_end = d_begin + g.Dg < L.D ? d_begin + g.Dg : L.D;
    const int32_t nb = g.nb;   // nb * P / 4 <= kProfPF * kNT
    const int64_t tile_n = g.A - a0 < kNT * kAPT ? g.A - a0 : kNT * kAPT;

    ProfArrivals<kAPT> s;
    {
        int32_t rp[kAPT], rU[kAPT];
        fetch_arrivals<kAPT>(g, a0, rp, rU);
        check_arrivals<kAPT>(g, group_max(V, d_begin, d_end).tot, rp, rU, s.p, s.U);
    }
#pragma unroll
    for (int k = 0; k < kAPT; ++k) {
        const int32_t U = s.U[k];
        s.neg[k] = U < 0 ? -1 : 0;
        s.off[k] = 4u * uint32_t(U < 0 ? 0 : (U < L.u_max ? U : L.u_max));
        s.best_key[k] = INT32_MAX;
        s.best_d[k] = d_begin;
    }

    DecLanes lanes = load_lanes(g, V, d_begin, d_end);
    int32_t lanes0 = d_begin;
    v4i stage[kProfPF];
    if (d_begin < d_end) {
        const int32_t n0 = d_end - d_begin < nb ? d_end - d_begin : nb;
        stage_profile(stage, V.prof, P, d_begin, n0 * (P / 4));
    }
    for (int32_t db = d_begin; db < d_end; db += nb) {
        const int32_t n = d_end - db < nb ? d_end - db : nb;
        const int32_t units = n * (P / 4);
        __syncthreads();   // every wave finished reading the previous batch
#pragma unroll
        for (int j = 0; j < kProfPF; ++j)
            if (j * kNT < units) reinterpret_cast<v4i*>(lds)[int(threadIdx.x) + j * kNT] = stage[j];
        __syncthreads();
        if (db + nb < d_end) {
            const int32_t n1 = d_end - (db + nb) < nb ? d_end - (db + nb) : nb;
            stage_profile(stage, V.prof, P, db + nb, n1 * (P / 4));   // overlaps the evaluation below
        }
        for (int32_t i = 0; i < n; ++i) {
            const int32_t d = db + i;
            if (d - lanes0 == kWave) {
                lanes = load_lanes(g, V, d, d_end);
                lanes0 = d;
            }
            const int32_t base = lane_value(lanes.base, d - lanes0);
            const int32_t C = lane_value(lanes.C, d - lanes0), Q = lane_value(lanes.Q, d - lanes0);
            if (threadIdx.x == 0 && (C < 0 || Q < 0)) raise_error(g.dev_err, MAPS_ERR_NEG_LEN);
            if (threadIdx.x == 0 && base < 0) raise_error(g.dev_err, MAPS_ERR_SNAPSHOT);
            const char* table = reinterpret_cast<const char*>(lds) + size_t(i) * P * 4;
            const __amdgpu_buffer_rsrc_t row = buffer_rsrc(kPairs ? g.pair + int64_t(d) * g.A + a0 : nullptr,
                                                           kPairs ? uint32_t(tile_n) * 4u : 0u);
            prof_decoder<kAPT, kFull, kPairs, kPolicy>(s, table, base, C, Q, d, row);
        }
    }
    write_partials<kAPT, kFull>(g, grp, a0, s.best_key, s.best_d);
}

template <int kAPT, bool kPairs, int kPolicy>
__global__ __launch_bounds__(kNT) void place_prof(PlaceArgs g) {
    extern __shared__ int4 lds[];
    const SnapView V = snap_view(const_cast<void*>(g.snap), g.L);
    if (!snapshot_ok(V.hdr, g.L)) {
        if (blockIdx.x == 0 && threadIdx.x == 0) raise_error(g.dev_err, MAPS_ERR_SNAPSHOT);
        return;
    }
    const int32_t grp = blockIdx.x % g.G;
    const int64_t a0 = int64_t(blockIdx.x / g.G) * (kNT * kAPT);
    if (a0 + kNT * kAPT <= g.A)
        prof_tile<kAPT, true, kPairs, kPolicy>(g, V, lds, grp, a0);
    else
        prof_tile<kAPT, false, kPairs, kPolicy>(g, V, lds, grp, a0);
}

// ---------------------------------------------------------------------------
// Final choice per arrival: the best group in group order (strictly smaller
// key wins, so ties keep the lower decoder), the chosen pair's peak, and the
// outputs; an arrival without a bound goes round-robin.  A key made from the
// overflow v = peak - C (policy MC, and MQ without a feasible decoder) gives
// the peak back; a feasible MQ choice evaluates its pair once more from the
// snapshot's records.
// ---------------------------------------------------------------------------
// The final selection for arrivals first, first + stride, ...  `scap`
// (nullable): LDS for the D capacities, staged by the workgroup while its
// first arrival's keys are on their way; every thread of the workgroup calls
// this with the same stride.
__device__ inline void finish_arrivals(const PlaceArgs& g, int64_t first, int64_t stride, int32_t* scap) {
    const SnapLayout& L = g.L;
    const SnapView V = snap_view(const_cast<void*>(g.snap), L);
    const int32_t ucl_max = 32 * L.W - 1;
    // the first arrival's bound and keys go out before anything that waits
    int32_t U = first < g.A ? g.aU[first] : -1;
    int32_t keys[kMaxGroups];
#pragma unroll
    for (int gi = 0; gi < kMaxGroups; ++gi)
        keys[gi] = first < g.A && gi < g.G ? g.pkey[int64_t(gi) * g.A + first] : INT32_MAX;
    if (!snapshot_ok(V.hdr, L)) return;   // uniform
    const int64_t n_total = load_uniform(&V.hdr->n_total);
    const int32_t* cap = g.cap;
    if (scap != nullptr) {
        for (int32_t d = threadIdx.x; d < L.D; d += blockDim.x) scap[d] = g.cap[d];
        __syncthreads();
        cap = scap;
    }
    for (int64_t a = first; a < g.A; a += stride) {
        if (a != first) {
            U = g.aU[a];
#pragma unroll
            for (int gi = 0; gi < kMaxGroups; ++gi) keys[gi] = gi < g.G ? g.pkey[int64_t(gi) * g.A + a] : INT32_MAX;
        }
        if (U < 0) {
            g.choice[a] = int32_t((g.rr_offset + a) % L.D);
            g.chosen_peak[a] = -1;
            g.chosen_over[a] = 0;
            g.flags[a] = 2;
            continue;
        }
        int32_t key = keys[0], best = 0;
#pragma unroll
        for (int gi = 1; gi < kMaxGroups; ++gi)
            if (keys[gi] < key) { key = keys[gi]; best = gi; }
        const int64_t od = int64_t(best) * g.A + a;
        int32_t d = g.dec16 ? int32_t(reinterpret_cast<const uint16_t*>(g.pdec)[od]) : g.pdec[od];
        d = d < 0 || d >= L.D ? 0 : d;
        const int32_t C = cap[d];
        int32_t peak = 0;
        if (g.policy == MAPS_POLICY_MC) {
            peak = int32_t(key_peak<MAPS_POLICY_MC>(key, C));
        } else if (key >= 0) {
            peak = int32_t(key_peak<MAPS_POLICY_MQ>(key, C));
        } else {
            const DecHeader h = V.dec[d];
            if (slice_ok(h, n_total, L)) {
                const int32_t p = g.ap[a] < 0 ? 0 : g.ap[a];
                const int32_t uc = U < ucl_max ? U : ucl_max;
                const uint2 w = slice_rank(V, h)[uc >> 5];
                uint32_t e = w.y + __popc(w.x & ((1u << (uc & 31)) - 1u));
                e = e < uint32_t(h.E) ? e : uint32_t(h.E);
                peak = event_peak(slice_pmx(V, h, L), slice_thr(V, h, L), slice_cold(V, h, L), e, p, U, h.base_peak);
            }
        }
        g.choice[a] = d;
        g.chosen_peak[a] = peak;
        g.chosen_over[a] = peak > C ? peak - C : 0;
        g.flags[a] = peak <= C ? 1 : 0;
    }
}

// Capacities staged in LDS for up to kFinishLdsDecoders decoders.
constexpr int32_t kFinishLdsDecoders = 16384;

__global__ __launch_bounds__(256) void place_finish(PlaceArgs g) {
    extern __shared__ int32_t scap[];
    finish_arrivals(g, int64_t(blockIdx.x) * blockDim.x + threadIdx.x, int64_t(gridDim.x) * blockDim.x,
                    g.L.D <= kFinishLdsDecoders ? scap : nullptr);
}

// The end of placement and every decoder's local order in one launch:
// workgroups [0, D) order one local queue each (dispatched first: they are
// the longer, latency-bound ones), the others make the final selection.  The
// two read the same snapshot and write disjoint outputs, so the selection
// runs beside the queue work.
__global__ __launch_bounds__(order::kOrderNT) void place_finish_order(PlaceArgs g, order::LocalArgs o,
                                                                      int32_t fin_blocks) {
    const int32_t D = o.L.D;
    if (int32_t(blockIdx.x) < D)
        order::order_queue(o, int32_t(blockIdx.x));
    else
        finish_arrivals(g, int64_t(int32_t(blockIdx.x) - D) * order::kOrderNT + threadIdx.x,
                        int64_t(fin_blocks) * order::kOrderNT, nullptr);
}

// ---------------------------------------------------------------------------
// Launch
// ---------------------------------------------------------------------------
template <int kAPT, bool kPairs, int kPolicy>
void launch_one(bool prof, dim3 grid, size_t lds, hipStream_t s, const PlaceArgs& a) {
    if (prof) {
        if constexpr (kAPT <= 8) {   // the profile path stages 64 VGPRs per thread
            auto fn = place_prof<kAPT, kPairs, kPolicy>;
            allow_dynamic_lds(fn, kLdsBytes);
            hipLaunchKernelGGL(fn, grid, dim3(kNT), lds, s, a);
        }
    } else {
        auto fn = place_records<kAPT, kPairs, kPolicy>;
        allow_dynamic_lds(fn, kLdsBytes);
        hipLaunchKernelGGL(fn, grid, dim3(kNT), lds, s, a);
    }
}

template <int kAPT>
void launch_apt(bool prof, bool pairs, int32_t policy, dim3 grid, size_t lds, hipStream_t s, const PlaceArgs& a) {
    if (pairs) {
        if (policy == MAPS_POLICY_MQ) launch_one<kAPT, true, MAPS_POLICY_MQ>(prof, grid, lds, s, a);
        else launch_one<kAPT, true, MAPS_POLICY_MC>(prof, grid, lds, s, a);
    } else {
        if (policy == MAPS_POLICY_MQ) launch_one<kAPT, false, MAPS_POLICY_MQ>(prof, grid, lds, s, a);
        else launch_one<kAPT, false, MAPS_POLICY_MC>(prof, grid, lds, s, a);
    }
}

// Arrivals per thread and decoder groups: the largest arrival tile (up to
// max_apt per thread) that still gives at least one workgroup per compute unit.
void plan(int32_t D, int64_t A, int cus, int max_apt, int* apt, int* groups) {
    for (int t : {16, 8, 4, 2, 1}) {
        if (t > max_apt) continue;
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
    int32_t* key;
    int32_t* dec;
    size_t bytes;
};

PlaceWorkspace place_carve(void* base, int64_t A) {
    PlaceWorkspace w;
    char* p = static_cast<char*>(base);
    size_t off = 0;
    auto take = [&](size_t bytes) { char* r = p ? p + off : nullptr; off += align256(bytes); return r; };
    w.key = reinterpret_cast<int32_t*>(take(size_t(kMaxGroups) * A * 4));
    w.dec = reinterpret_cast<int32_t*>(take(size_t(kMaxGroups) * A * 4));
    w.bytes = off;
    return w;
}

}  // namespace
}  // namespace maps

using namespace maps;

extern "C" size_t maps_place_workspace_size(int32_t D, int64_t A, int32_t u_max) {
    if (D < 1 || A < 0 || u_max < 0) return 0;
    return place_carve(nullptr, A).bytes;
}

namespace {

// Checks the arguments of a placement and, when A > 0, launches its records
// pass and fills *out for the final selection (*launched = A > 0).
maps_status place_records_enqueue(const void* snapshot, int32_t D, int32_t u_max, const int32_t* capacity,
                                  const int32_t* queue_len, const int32_t* a_prompt, const int32_t* a_upper,
                                  int64_t A, int32_t policy, int64_t rr_offset, int32_t* choice,
                                  int32_t* chosen_peak, int32_t* chosen_overflow, uint8_t* flags,
                                  int32_t* pair_peak, uint32_t* dev_err, void* workspace,
                                  size_t workspace_bytes, hipStream_t stream, PlaceArgs* out, bool* launched) {
    *launched = false;
    if (D < 1 || A < 0 || rr_offset < 0 || u_max < 0 || u_max > MAPS_MAX_U_MAX) return MAPS_E_SIZE;
    if (policy != MAPS_POLICY_MQ && policy != MAPS_POLICY_MC) return MAPS_E_POLICY;
    if (!snapshot || !capacity || !queue_len || !dev_err ||
        (A > 0 && (!a_prompt || !a_upper || !choice || !chosen_peak || !chosen_overflow || !flags)))
        return MAPS_E_NULL;
    if (A == 0) return MAPS_OK;
    if (!workspace) return MAPS_E_NULL;
    const PlaceWorkspace w = place_carve(workspace, A);
    if (workspace_bytes < w.bytes) return MAPS_E_WORKSPACE;
    const SnapLayout L = snap_layout(D, 0, u_max);   // region offsets do not depend on the resident count
    const bool prof = L.P > 0;
    int apt = 8, G = 1;
    plan(D, A, device_compute_units(), prof ? 8 : 16, &apt, &G);
    PlaceArgs a{};
    a.L = L;
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
    a.dec16 = D <= 65536;
    a.G = G;
    a.policy = policy;
    a.Dg = (D + G - 1) / G;
    a.dev_err = dev_err;
    // Slices are addressed through the decoder headers and bound-checked
    // against the snapshot's own resident count.
    size_t lds = 0;
    if (prof) {
        // LDS: the staged units of one batch of nb profiles
        const int64_t nb = int64_t(kProfPF) * kNT * 4 / L.P;
        a.nb = int32_t(nb < 8 ? nb : 8);
        lds = size_t(kProfPF) * kNT * 16;
    } else {
        // two buffers of kStage * kNT 16-byte units: the staged part of a slice
        const int32_t buf_units = kStage * kNT;
        a.buf_units = L.W / 2 + 64 <= buf_units ? buf_units : 0;
        lds = size_t(2 * a.buf_units) * 16 + kRedBytes;
    }
    const int64_t tiles = (A + int64_t(kNT) * apt - 1) / (int64_t(kNT) * apt);
    const dim3 grid(unsigned(tiles * G));
    const bool pairs = pair_peak != nullptr;
    switch (apt) {
        case 16: launch_apt<16>(prof, pairs, policy, grid, lds, stream, a); break;
        case 8: launch_apt<8>(prof, pairs, policy, grid, lds, stream, a); break;
        case 4: launch_apt<4>(prof, pairs, policy, grid, lds, stream, a); break;
        case 2: launch_apt<2>(prof, pairs, policy, grid, lds, stream, a); break;
        default: launch_apt<1>(prof, pairs, policy, grid, lds, stream, a); break;
    }
    MAPS_CHECK_LAUNCH();
    *out = a;
    *launched = true;
    return MAPS_OK;
}

}  // namespace

extern "C" maps_status maps_place(const void* snapshot, int32_t D, int32_t u_max, const int32_t* capacity,
                                  const int32_t* queue_len, const int32_t* a_prompt, const int32_t* a_upper,
                                  int64_t A, int32_t policy, int64_t rr_offset, int32_t* choice,
                                  int32_t* chosen_peak, int32_t* chosen_overflow, uint8_t* flags,
                                  int32_t* pair_peak, uint32_t* dev_err, void* workspace,
                                  size_t workspace_bytes, hipStream_t stream) {
    PlaceArgs a{};
    bool launched = false;
    const maps_status st = place_records_enqueue(snapshot, D, u_max, capacity, queue_len, a_prompt, a_upper, A,
                                                 policy, rr_offset, choice, chosen_peak, chosen_overflow, flags,
                                                 pair_peak, dev_err, workspace, workspace_bytes, stream, &a,
                                                 &launched);
    if (st != MAPS_OK || !launched) return st;
    const int64_t blocks = (A + 255) / 256;
    const size_t lds = D <= kFinishLdsDecoders ? size_t(D) * sizeof(int32_t) : 0;
    allow_dynamic_lds(place_finish, lds);
    hipLaunchKernelGGL(place_finish, dim3(unsigned(blocks < 4096 ? blocks : 4096)), dim3(256), lds, stream, a);
    MAPS_CHECK_LAUNCH();
    return MAPS_OK;
}

extern "C" maps_status maps_place_order(const void* snapshot, int32_t D, int32_t u_max, const int32_t* capacity,
                                        const int32_t* queue_len, const int32_t* a_prompt, const int32_t* a_upper,
                                        int64_t A, int32_t policy, int64_t rr_offset, int32_t* choice,
                                        int32_t* chosen_peak, int32_t* chosen_overflow, uint8_t* flags,
                                        int32_t* pair_peak, const int64_t* q_off, int64_t q_total,
                                        const int32_t* q_prompt, const int32_t* q_upper, const int32_t* q_wait_ms,
                                        int32_t max_wait_ms, int32_t* order, int32_t* admitted, uint32_t* dev_err,
                                        void* workspace, size_t workspace_bytes, hipStream_t stream) {
    // the local-order arguments first: nothing is enqueued when either set is wrong
    if (D < 1 || q_total < 0 || u_max < 0 || u_max > MAPS_MAX_U_MAX) return MAPS_E_SIZE;
    if (!q_off || !admitted || (q_total > 0 && (!q_prompt || !q_upper || !order))) return MAPS_E_NULL;
    if (D < 1 || A < 0 || rr_offset < 0) return MAPS_E_SIZE;
    if (policy != MAPS_POLICY_MQ && policy != MAPS_POLICY_MC) return MAPS_E_POLICY;
    if (!snapshot || !capacity || !queue_len || !dev_err ||
        (A > 0 && (!a_prompt || !a_upper || !choice || !chosen_peak || !chosen_overflow || !flags)) ||
        (A > 0 && !workspace))
        return MAPS_E_NULL;
    if (A > 0 && workspace_bytes < place_carve(nullptr, A).bytes) return MAPS_E_WORKSPACE;
    PlaceArgs a{};
    bool launched = false;
    const maps_status st = place_records_enqueue(snapshot, D, u_max, capacity, queue_len, a_prompt, a_upper, A,
                                                 policy, rr_offset, choice, chosen_peak, chosen_overflow, flags,
                                                 pair_peak, dev_err, workspace, workspace_bytes, stream, &a,
                                                 &launched);
    if (st != MAPS_OK) return st;
    order::LocalArgs o;
    o.L = snap_layout(D, 0, u_max);
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
    int64_t fin = launched ? (A + order::kOrderNT - 1) / order::kOrderNT : 0;
    fin = fin < 1024 ? fin : 1024;
    hipLaunchKernelGGL(place_finish_order, dim3(unsigned(fin + D)), dim3(order::kOrderNT), 0, stream, a, o,
                       int32_t(fin));
    MAPS_CHECK_LAUNCH();
    return MAPS_OK;
}
