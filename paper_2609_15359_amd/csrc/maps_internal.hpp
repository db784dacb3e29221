// Internal definitions of the MAPS scheduler core for gfx950: the snapshot
// layout shared by projection, placement and local ordering, launch helpers and
// workgroup-wide scans.  Not part of the public ABI (see include/maps.h).
#pragma once

#include <hip/hip_runtime.h>
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
// Record e (0 <= e <= E) stores {PMX_e, S_e, N_e + 1, tau_e}; record E is
// {PMX_E, 0, 1, INT32_MAX}.  The rank e = #{events < U} comes from a bitmap
// over the step axis: word w holds bit j for event time 32w + j, next to the
// number of events before word w.  W words cover [0, 32 W) with 32 W - 1 > u_max,
// so a bound clamped to 32 W - 1 ranks above every event.
// ---------------------------------------------------------------------------
struct SnapHeader {       // at offset 0, 64 bytes
    uint32_t magic;
    int32_t D;
    int32_t u_max;
    int32_t W;            // rank words per decoder
    int64_t n_total;      // residents
    int64_t max_tot;      // max over decoders of sum_r (p + g + R)
    int32_t max_records;  // max over decoders of E + 1
    int32_t pad[7];
};
static_assert(sizeof(SnapHeader) == 64, "header size");

struct DecHeader {        // one per decoder, 32 bytes
    int64_t rec_off;      // index of record 0 of this decoder
    int64_t tot;          // sum_r (p + g + R)
    int32_t E;            // number of events
    int32_t base_peak;    // max_t O(t)
    int32_t pad[2];
};
static_assert(sizeof(DecHeader) == 32, "decoder header size");

// Rank words per decoder: 32 W - 1 > u_max, rounded up to an even count so each
// decoder's slice starts on a 16-byte boundary.
__host__ __device__ inline int32_t rank_words(int32_t u_max) { return (((u_max + 1) / 32 + 1) + 1) & ~1; }

struct SnapLayout {
    int32_t D, u_max, W;
    int64_t n_total;
    size_t off_dec, off_rank, off_rec, bytes;
};

__host__ __device__ inline SnapLayout snap_layout(int32_t D, int64_t n_total, int32_t u_max) {
    SnapLayout L;
    L.D = D;
    L.u_max = u_max;
    L.W = rank_words(u_max);
    L.n_total = n_total;
    L.off_dec = align256(sizeof(SnapHeader));
    L.off_rank = L.off_dec + align256(size_t(D) * sizeof(DecHeader));
    L.off_rec = L.off_rank + align256(size_t(D) * size_t(L.W) * sizeof(uint2));
    // 64 spare records at the end: placement copies records in transfers of
    // 64, so it reads up to 63 records past a decoder's last one
    L.bytes = L.off_rec + size_t(n_total + D + 64) * sizeof(int4);
    return L;
}

struct SnapView {
    SnapHeader* hdr;
    DecHeader* dec;
    uint2* rank;   // [D][W] {bits, events before the word}
    int4* rec;     // records {PMX, S, N+1, tau}
};

__host__ __device__ inline SnapView snap_view(void* base, const SnapLayout& L) {
    char* b = static_cast<char*>(base);
    return SnapView{reinterpret_cast<SnapHeader*>(b), reinterpret_cast<DecHeader*>(b + L.off_dec),
                    reinterpret_cast<uint2*>(b + L.off_rank), reinterpret_cast<int4*>(b + L.off_rec)};
}

// ---------------------------------------------------------------------------
// Device helpers
// ---------------------------------------------------------------------------
__device__ inline void raise_error(uint32_t* dev_err, uint32_t bits) {
    if (dev_err) atomicOr(dev_err, bits);
}

template <typename T>
__device__ inline T wave_incl_scan_add(T v) {
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        T o = __shfl_up(v, off, kWave);
        if (int(threadIdx.x % kWave) >= off) v += o;
    }
    return v;
}

template <typename T>
__device__ inline T wave_incl_scan_max(T v) {
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        T o = __shfl_up(v, off, kWave);
        if (int(threadIdx.x % kWave) >= off) v = v > o ? v : o;
    }
    return v;
}

template <typename T>
__device__ inline T wave_reduce_add(T v) {
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) v += __shfl_xor(v, off, kWave);
    return v;
}

template <typename T>
__device__ inline T wave_reduce_max(T v) {
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) {
        T o = __shfl_xor(v, off, kWave);
        v = v > o ? v : o;
    }
    return v;
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
// thread's exclusive prefix and writes the total to *total.
template <int NT, bool kMax, typename T>
__device__ inline T block_excl_scan(T v, T identity, T* tmp, T* total) {
    const int lane = threadIdx.x % kWave, wid = threadIdx.x / kWave;
    T incl = kMax ? wave_incl_scan_max(v) : wave_incl_scan_add(v);
    __syncthreads();
    if (lane == kWave - 1) tmp[wid] = incl;
    __syncthreads();
    T wave_prefix = identity, all = identity;
#pragma unroll
    for (int i = 0; i < NT / kWave; ++i) {
        T x = tmp[i];
        if (i < wid) wave_prefix = kMax ? (wave_prefix > x ? wave_prefix : x) : wave_prefix + x;
        all = kMax ? (all > x ? all : x) : all + x;
    }
    T excl_in_wave = __shfl_up(incl, 1, kWave);
    if (lane == 0) excl_in_wave = identity;
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
template <typename Kernel>
inline void allow_dynamic_lds(Kernel* fn, size_t bytes) {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(fn), hipFuncAttributeMaxDynamicSharedMemorySize,
                              int(bytes));
}

}  // namespace maps

// Host-side launch check: returns MAPS_E_HIP from the enclosing function when
// the last launch failed.
#define MAPS_CHECK_LAUNCH()                                  \
    do {                                                     \
        if (hipGetLastError() != hipSuccess) return MAPS_E_HIP; \
    } while (0)
