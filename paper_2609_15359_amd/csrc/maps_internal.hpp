// Internal definitions of the MAPS scheduler core for gfx950: the snapshot
// layout shared by projection, placement and local ordering, launch helpers and
// workgroup-wide scans.  Not part of the public ABI (see include/maps.h).
#pragma once

#include <hip/hip_runtime.h>
#include <limits>
#include <stdint.h>

#include "maps.h"

namespace maps {

constexpr uint32_t kSnapMagic = 0x5350414Du;  // "MAPS"
constexpr int kWave = 64;                     // CDNA wavefront width

__host__ __device__ inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// ---------------------------------------------------------------------------
// Snapshot of the projected occupancy of D decoders.
//
// For decoder d with resident remaining lengths R_r = max(U_r - g_r, 0), let
// tau_0 < tau_1 < ... < tau_{E-1} be the distinct values of R_r (the events),
// N_e = #{r : R_r >= tau_e} and S_e = sum_{R_r >= tau_e} (p_r + g_r).  Between
// events the active set is constant, so on (tau_{e-1}, tau_e] the occupancy is
// O(t) = S_e + t N_e, increasing in t; O(t) = 0 after tau_{E-1}.
//
// An arrival with bound U and prompt p is present at the steps t <= U, where
// O(t) + p + t is increasing inside each event interval, so
//   PF(U) = max_{t <= U} (O(t) + t) = max(PMX_e, S_e + U (N_e + 1)),
//   e = #{events < U},   PMX_e = max(0, max_{i < e} S_i + tau_i (N_i + 1)),
// with S_E = N_E = 0 for e = E.  The steps after U contribute at most
// base = max_t O(t); and if U reaches the first step of maximal occupancy,
// PF(U) >= base already.  Hence the projected peak with the arrival is
//   peak(p, U) = max(p + PF(U), base).
//
// Each event e (0 <= e <= E, with S_E = N_E = 0) has
//   PMX_e, and T_e = the smallest U with S_e + U (N_e + 1) > PMX_e
//          (0 when S_e > PMX_e; capped at INT32_MAX), in two int32 arrays,
//   and the cold record {S_e, N_e + 1}.
// For U < T_e, PF(U) = PMX_e and the cold record is not needed; for U >= T_e,
// PF(U) = S_e + U (N_e + 1).  A bound lands on event e when tau_{e-1} < U <=
// tau_e, so the bounds that need a cold record form the ranges
// [max(T_e, tau_{e-1} + 1), tau_e] for e < E (at e = E, S = N = 0 and
// max(PMX_E, U) is exact); the header's hot window [hot_lo, hot_hi] lies above
// event 0's range and below every later one.  PMX_e is nondecreasing: once it
// reaches PMX_E (at event e*), every bound U >= flat_lo = tau_{e*-1} + 1 that
// lies in the hot window has PF(U) = max(PMX_E, U), with no lookup at all.  The rank e = #{events < U} comes from a bitmap
// over the step axis: word w holds bit j for event time 32w + j, next to the
// number of events before word w.  W words cover [0, 32 W) with 32 W - 1 > u_max,
// so a bound clamped to 32 W - 1 ranks above every event.  Each decoder's rank
// words and event data form one contiguous slice of 16-byte units: W/2 units
// of rank words, the E + 1 PMX values and the E + 1 thresholds (each array
// padded to whole units), then the E + 1 cold records; a consumer copies the
// prefix it needs in one pass.
//
// Since PF depends on the arrival only through U, a decoder whose bounds are
// short enough also gets a dense profile F(u) = max(PF(u), u) for u = 0..u_max
// (P >= u_max + 1 entries, the tail padded with the same formula).  For any
// U >= 0, F(min(U, u_max)) and U give PF exactly: F(u) >= u, and beyond u_max
// no event remains, so PF(U) = max(F(u_max), U).  Placement then needs one
// table read per pair:  peak(p, U) = max(p + max(F(min(U, u_max)), U), base).
// ---------------------------------------------------------------------------
struct SnapHeader {       // at offset 0, 64 bytes
    uint32_t magic;
    int32_t D;
    int32_t u_max;
    int32_t W;            // rank words per decoder
    int64_t n_total;      // residents
    int32_t P;            // profile entries per decoder (0: no profile)
    int32_t pad[9];
};
static_assert(sizeof(SnapHeader) == 64, "header size");

struct DecHeader {        // one per decoder, 64 bytes
    int64_t slice_off;    // first 16-byte unit of this decoder's slice
    int64_t tot;          // sum_r (p + g + R)
    int32_t E;            // number of events
    int32_t base_peak;    // max_t O(t)
    int32_t hot_lo;       // every bound U in [hot_lo, hot_hi] has PF(U) = max(PMX_e, U):
    int32_t hot_hi;       //   it stays below the threshold of the event it lands on
    int32_t flat_lo;      // every bound U >= flat_lo lands on an event e with PMX_e = PMX_E
    int32_t pmx_end;      // PMX_E, the largest S_e + tau_e (N_e + 1)
    int32_t pad[6];
};
static_assert(sizeof(DecHeader) == 64, "decoder header size");

// Rank words per decoder: 32 W - 1 > u_max, rounded up to an even count so each
// decoder's slice starts on a 16-byte boundary.
__host__ __device__ inline int32_t rank_words(int32_t u_max) { return (((u_max + 1) / 32 + 1) + 1) & ~1; }

// Profile entries per decoder: u_max + 1 rounded up to a multiple of 4 (whole
// 16-byte units), or 0 when the table would exceed kProfileMaxEntries.  The
// rank words cover every padded entry: 32 W >= round_up(u_max + 1, 32) >= P.
constexpr int32_t kProfileMaxEntries = 16384;
__host__ __device__ inline int32_t profile_entries(int32_t u_max) {
    return u_max + 1 <= kProfileMaxEntries ? (u_max + 4) & ~3 : 0;
}

struct SnapLayout {
    int32_t D, u_max, W, P;
    int64_t n_total;
    size_t off_dec, off_prof, off_slice, bytes;
};

// 16-byte units of one int32 array over the events 0..E.
__host__ __device__ inline int64_t event_units(int64_t E) { return (E + 4) / 4; }

// Units of a decoder's slice with E events: rank words, PMX, T, cold records.
// With E <= n_d residents this is at most W/2 + n_d + kSliceSpare.
constexpr int kSliceSpare = 3;
__host__ __device__ inline int64_t slice_span(int32_t W, int64_t E) {
    return W / 2 + 2 * event_units(E) + (E + 2) / 2;
}

// Units of the slice region: n_total, plus W/2 + kSliceSpare per decoder.
__host__ __device__ inline int64_t slice_units(const SnapLayout& L) {
    return L.n_total + int64_t(L.D) * (kSliceSpare + L.W / 2);
}

__host__ __device__ inline SnapLayout snap_layout(int32_t D, int64_t n_total, int32_t u_max) {
    SnapLayout L;
    L.D = D;
    L.u_max = u_max;
    L.W = rank_words(u_max);
    L.P = profile_entries(u_max);
    L.n_total = n_total;
    L.off_dec = align256(sizeof(SnapHeader));
    L.off_prof = L.off_dec + align256(size_t(D) * sizeof(DecHeader));
    L.off_slice = L.off_prof + align256(size_t(D) * size_t(L.P) * sizeof(int32_t));
    // decoder d with residents [lo, hi) owns the units [lo + d s, hi + (d + 1) s), s = kSliceSpare + W/2;
    // 64 spare units at the end
    L.bytes = L.off_slice + size_t(slice_units(L) + 64) * sizeof(int4);
    return L;
}

struct SnapView {
    SnapHeader* hdr;
    DecHeader* dec;
    int4* slices;   // per decoder: W/2 units of rank words {bits, events before the word}, then
                    // PMX[E + 1], T[E + 1] and the cold records {S, N + 1}[E + 1]
    int32_t* prof;  // [D][P] profile F(u)
};

__host__ __device__ inline SnapView snap_view(void* base, const SnapLayout& L) {
    char* b = static_cast<char*>(base);
    return SnapView{reinterpret_cast<SnapHeader*>(b), reinterpret_cast<DecHeader*>(b + L.off_dec),
                    reinterpret_cast<int4*>(b + L.off_slice), reinterpret_cast<int32_t*>(b + L.off_prof)};
}

// Whether a decoder header describes a slice inside the snapshot (n_total
// from the snapshot's own header).
__host__ __device__ inline bool slice_ok(const DecHeader& h, int64_t n_total, const SnapLayout& L) {
    return h.E >= 0 && h.slice_off >= 0 && h.base_peak >= 0 &&
           h.slice_off + slice_span(L.W, h.E) <= n_total + int64_t(L.D) * (kSliceSpare + L.W / 2);
}
__host__ __device__ inline const uint2* slice_rank(const SnapView& V, const DecHeader& h) {
    return reinterpret_cast<const uint2*>(V.slices + h.slice_off);
}
__host__ __device__ inline const int32_t* slice_pmx(const SnapView& V, const DecHeader& h, const SnapLayout& L) {
    return reinterpret_cast<const int32_t*>(V.slices + h.slice_off + L.W / 2);
}
__host__ __device__ inline const int32_t* slice_thr(const SnapView& V, const DecHeader& h, const SnapLayout& L) {
    return slice_pmx(V, h, L) + 4 * event_units(h.E);
}
__host__ __device__ inline const int2* slice_cold(const SnapView& V, const DecHeader& h, const SnapLayout& L) {
    return reinterpret_cast<const int2*>(V.slices + h.slice_off + L.W / 2 + 2 * event_units(h.E));
}

// Threshold T of an event: the smallest U >= 0 with S + U n1 > pmx.
__host__ __device__ inline int32_t event_threshold(int32_t pmx, int32_t S, uint32_t n1) {
    if (S > pmx) return 0;
    const int32_t diff = pmx - S;
    if (diff >= 0) {   // every valid snapshot: a 32-bit division
        const uint32_t q = uint32_t(diff) / n1;
        return q < uint32_t(INT32_MAX - 1) ? int32_t(q + 1) : INT32_MAX;
    }
    const int64_t t = int64_t(diff) / int64_t(n1) + 1;
    return t < int64_t(INT32_MAX) ? int32_t(t) : INT32_MAX;
}

// ---------------------------------------------------------------------------
// Device helpers
// ---------------------------------------------------------------------------
__device__ inline void raise_error(uint32_t* dev_err, uint32_t bits) {
    if (dev_err) atomicOr(dev_err, bits);
}

// Wavefront scans and reductions through DPP (data-parallel primitives: a
// lane reads another lane's register as an instruction operand, no LDS
// round trip).  The inclusive scan is Hillis-Steele within each row of 16
// lanes (row shifts by 1, 2, 4, 8), then the row broadcasts of gfx9: lane 15
// of rows 0 and 2 into rows 1 and 3, then lane 31 into rows 2 and 3.  Lanes
// without a source keep `fill`, the operation's identity.  Called by whole
// wavefronts.
constexpr int kDppRowShr1 = 0x111, kDppRowShr2 = 0x112, kDppRowShr4 = 0x114, kDppRowShr8 = 0x118;
constexpr int kDppWaveShr1 = 0x138, kDppRowBcast15 = 0x142, kDppRowBcast31 = 0x143;

template <int kCtrl, int kRowMask, typename T>
__device__ inline T dpp_move(T fill, T v) {
    static_assert(sizeof(T) == 4 || sizeof(T) == 8, "32- or 64-bit values");
    if constexpr (sizeof(T) == 4) {
        return __builtin_bit_cast(T, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, fill),
                                                                 __builtin_bit_cast(int, v), kCtrl, kRowMask,
                                                                 0xf, false));
    } else {
        const uint64_t f = __builtin_bit_cast(uint64_t, fill), x = __builtin_bit_cast(uint64_t, v);
        const uint32_t lo = uint32_t(__builtin_amdgcn_update_dpp(int(uint32_t(f)), int(uint32_t(x)), kCtrl,
                                                                 kRowMask, 0xf, false));
        const uint32_t hi = uint32_t(__builtin_amdgcn_update_dpp(int(uint32_t(f >> 32)), int(uint32_t(x >> 32)),
                                                                 kCtrl, kRowMask, 0xf, false));
        return __builtin_bit_cast(T, (uint64_t(hi) << 32) | lo);
    }
}

template <typename T, typename Op>
__device__ inline T wave_incl_scan(T v, T fill, Op op) {
    v = op(v, dpp_move<kDppRowShr1, 0xf>(fill, v));
    v = op(v, dpp_move<kDppRowShr2, 0xf>(fill, v));
    v = op(v, dpp_move<kDppRowShr4, 0xf>(fill, v));
    v = op(v, dpp_move<kDppRowShr8, 0xf>(fill, v));
    v = op(v, dpp_move<kDppRowBcast15, 0xa>(fill, v));
    v = op(v, dpp_move<kDppRowBcast31, 0xc>(fill, v));
    return v;
}

// The value of lane 63, in every lane.
template <typename T>
__device__ inline T wave_last(T v) {
    if constexpr (sizeof(T) == 4) {
        return __builtin_bit_cast(T, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), kWave - 1));
    } else {
        const uint64_t x = __builtin_bit_cast(uint64_t, v);
        const uint32_t lo = uint32_t(__builtin_amdgcn_readlane(int(uint32_t(x)), kWave - 1));
        const uint32_t hi = uint32_t(__builtin_amdgcn_readlane(int(uint32_t(x >> 32)), kWave - 1));
        return __builtin_bit_cast(T, (uint64_t(hi) << 32) | lo);
    }
}

// Lane i gets lane i - 1's value, lane 0 gets `fill`.
template <typename T>
__device__ inline T wave_shift_up1(T v, T fill) {
    return dpp_move<kDppWaveShr1, 0xf>(fill, v);
}

template <typename T>
__device__ inline T wave_incl_scan_add(T v) {
    return wave_incl_scan(v, T(0), [](T x, T y) { return x + y; });
}

template <typename T>
__device__ inline T wave_incl_scan_max(T v) {
    return wave_incl_scan(v, std::numeric_limits<T>::lowest(), [](T x, T y) { return x > y ? x : y; });
}

template <typename T>
__device__ inline T wave_reduce_add(T v) {
    return wave_last(wave_incl_scan_add(v));
}

template <typename T>
__device__ inline T wave_reduce_max(T v) {
    return wave_last(wave_incl_scan_max(v));
}

// Workgroup-wide reductions over one value per thread; `tmp` holds NT/64 slots.
template <int NT, typename T>
__device__ inline T block_reduce_add(T v, T* tmp) {
    v = wave_reduce_add(v);
    const int lane = threadIdx.x % kWave, wid = threadIdx.x / kWave;
    __syncthreads();
    if (lane == 0) tmp[wid] = v;
    __syncthreads();
    T s = 0;
#pragma unroll
    for (int i = 0; i < NT / kWave; ++i) s += tmp[i];
    return s;
}

template <int NT, typename T>
__device__ inline T block_reduce_max(T v, T* tmp) {
    v = wave_reduce_max(v);
    const int lane = threadIdx.x % kWave, wid = threadIdx.x / kWave;
    __syncthreads();
    if (lane == 0) tmp[wid] = v;
    __syncthreads();
    T s = tmp[0];
#pragma unroll
    for (int i = 1; i < NT / kWave; ++i) s = s > tmp[i] ? s : tmp[i];
    return s;
}

// Exclusive scan of one value per thread across the workgroup; returns the
// thread's exclusive prefix and writes the total to *total.  Without
// kGuard the caller guarantees that no thread still reads `tmp` from an
// earlier use (the leading barrier is skipped).
template <int NT, bool kMax, typename T, bool kGuard = true>
__device__ inline T block_excl_scan(T v, T identity, T* tmp, T* total) {
    const int lane = threadIdx.x % kWave, wid = threadIdx.x / kWave;
    T incl = kMax ? wave_incl_scan_max(v) : wave_incl_scan_add(v);
    if constexpr (kGuard) __syncthreads();
    if (lane == kWave - 1) tmp[wid] = incl;
    __syncthreads();
    T wave_prefix = identity, all = identity;
#pragma unroll
    for (int i = 0; i < NT / kWave; ++i) {
        T x = tmp[i];
        if (i < wid) wave_prefix = kMax ? (wave_prefix > x ? wave_prefix : x) : wave_prefix + x;
        all = kMax ? (all > x ? all : x) : all + x;
    }
    const T excl_in_wave = wave_shift_up1(incl, identity);
    *total = all;
    return kMax ? (wave_prefix > excl_in_wave ? wave_prefix : excl_in_wave) : wave_prefix + excl_in_wave;
}

// Scan of len elements reached through get(i)/put(i, v), each thread owning
// one contiguous chunk.  Forward or reverse (suffix), inclusive or exclusive,
// sum or max.  Returns the total.  Ends with a barrier.
template <int NT, bool kMax, bool kReverse, bool kExclusive, typename T, typename Get, typename Put>
__device__ inline T block_scan(int64_t len, T identity, Get get, Put put, T* tmp) {
    const int64_t chunk = (len + NT - 1) / NT;
    const int64_t b = int64_t(threadIdx.x) * chunk;
    const int64_t e = b + chunk < len ? b + chunk : len;
    auto idx = [&](int64_t i) { return kReverse ? len - 1 - i : i; };
    T acc = identity;
    for (int64_t i = b; i < e; ++i) {
        T x = get(idx(i));
        acc = kMax ? (acc > x ? acc : x) : acc + x;
    }
    T total;
    T run = block_excl_scan<NT, kMax>(acc, identity, tmp, &total);
    for (int64_t i = b; i < e; ++i) {
        T x = get(idx(i));
        T next = kMax ? (run > x ? run : x) : run + x;
        put(idx(i), kExclusive ? run : next);
        run = next;
    }
    __syncthreads();
    return total;
}

// Host: let a kernel use `bytes` of dynamic LDS (gfx950 has 160 KB per CU).
// Each kernel's attribute is set once per process, so that calls made while
// a stream is being captured into a graph issue no attribute change.
void allow_dynamic_lds_fn(const void* fn, size_t bytes);
template <typename Kernel>
inline void allow_dynamic_lds(Kernel* fn, size_t bytes) {
    allow_dynamic_lds_fn(reinterpret_cast<const void*>(fn), bytes);
}

// Host: compute units of the current device, queried once per device.
int device_compute_units();

// LDS of one workgroup on gfx950, static and dynamic together.
constexpr size_t kLdsPerWorkgroup = 160 * 1024;

// Host: a kernel's static LDS in bytes, queried once per kernel.
size_t kernel_static_lds(const void* fn);
template <typename Kernel>
inline size_t kernel_static_lds(Kernel* fn) {
    return kernel_static_lds(reinterpret_cast<const void*>(fn));
}

}  // namespace maps

// Host-side launch check: returns MAPS_E_HIP from the enclosing function when
// the last launch failed.
#define MAPS_CHECK_LAUNCH()                                  \
    do {                                                     \
        if (hipGetLastError() != hipSuccess) return MAPS_E_HIP; \
    } while (0)
