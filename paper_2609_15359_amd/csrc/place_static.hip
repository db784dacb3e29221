// Algorithm 1 on block counts (Sec. 3.3: the runtime state of each decoder,
// Eq. (6), Algorithm 1, and the atomic reservation of B_need after each
// dispatch) on gfx950.
//
//   rsc_state           one workgroup per decoder: held and reserved blocks of
//                       its residents (and of requests whose prompt KV is
//                       still in transfer) summed in 64-bit integers;
//   static_independent  every arrival against the reported state: the
//                       decoders' (B_eff, Q) staged in LDS in tiles, each
//                       thread scanning them for four arrivals at once (the
//                       LDS reads are broadcasts);
//   static_need         every arrival's B_need, in parallel;
//   static_reserve      arrivals one after another, each reserving its B_need
//                       and joining its decoder's queue before the next: one
//                       wavefront holds the state of up to 1,024 decoders in
//                       registers (ceil(D/64) per lane, a template parameter);
//                       the largest B_eff is kept from one arrival to the next
//                       (a wavefront maximum through DPP after each
//                       reservation), so an arrival that fits no decoder takes
//                       it directly; a feasible shortest-queue choice takes a
//                       wavefront minimum over every decoder.  The owning lane
//                       updates its register.  The chain is serial by
//                       definition, so this kernel runs at the latency of one
//                       wavefront.
#include <type_traits>

#include "maps_internal.hpp"

namespace maps {
namespace {

constexpr int kRscNT = 256;
constexpr int kIndNT = 256;
constexpr int kIndPer = 4;           // arrivals per thread
constexpr int kIndTile = 2048;       // decoders per LDS tile
constexpr int kResSlots = MAPS_MAX_RESERVE_DECODERS / kWave;
constexpr int64_t kBlockLimit = int64_t(1) << 52;

__device__ inline int64_t ceil_blocks(int64_t tokens, int64_t S) { return (tokens + S - 1) / S; }

// ---------------------------------------------------------------------------
// Runtime state
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kRscNT) void rsc_state(int32_t D, const int64_t* __restrict__ seg_off,
                                                    int64_t n_total, const int32_t* __restrict__ p,
                                                    const int32_t* __restrict__ g, const int32_t* __restrict__ U,
                                                    const uint8_t* __restrict__ in_flight,
                                                    const int32_t* __restrict__ cap, int32_t S,
                                                    int64_t* __restrict__ b_free, int64_t* __restrict__ b_res,
                                                    int64_t* __restrict__ b_eff, uint32_t* dev_err) {
    __shared__ int64_t tmp[kRscNT / kWave];
    const int d = blockIdx.x;
    int64_t lo = seg_off[d], hi = seg_off[d + 1];
    if (!(0 <= lo && lo <= hi && hi <= n_total)) {
        if (threadIdx.x == 0) {
            raise_error(dev_err, MAPS_ERR_SEG_OFFSETS);
            b_free[d] = b_res[d] = b_eff[d] = 0;
        }
        return;
    }
    int64_t held = 0, res = 0;
    bool bad = false;
    for (int64_t r = lo + threadIdx.x; r < hi; r += kRscNT) {
        const int32_t pr = p[r], gr = g[r], ur = U[r];
        if (in_flight && in_flight[r]) {
            // staged reservation: prompt KV still in transfer, nothing held,
            // the whole budget (the prompt's blocks without a bound) reserved
            bad |= pr < 0;
            res += ceil_blocks(int64_t(pr) + (ur < 0 ? 0 : ur), S);
            continue;
        }
        bad |= (pr < 0) | (gr < 0);
        const int64_t now = ceil_blocks(int64_t(pr) + gr, S);
        const int64_t demand = ur < 0 ? now : ceil_blocks(int64_t(pr) + ur, S);
        held += now;
        res += demand > now ? demand - now : 0;
    }
    if (bad) raise_error(dev_err, MAPS_ERR_NEG_LEN);
    held = block_reduce_add<kRscNT>(held, tmp);
    res = block_reduce_add<kRscNT>(res, tmp);
    if (threadIdx.x == 0) {
        const int32_t c = cap[d];
        if (c < 0) raise_error(dev_err, MAPS_ERR_NEG_LEN);
        const int64_t fr = int64_t(c) / S - held;
        b_free[d] = fr;
        b_res[d] = res;
        b_eff[d] = fr - res;
    }
}

struct StaticArgs {
    int32_t D;
    const int64_t* beff;
    const int32_t* qlen;
    int32_t S;
    const int32_t* ap;
    const int32_t* aU;
    int64_t A;
    int32_t policy;
    int64_t rr_offset;
    int32_t* choice;
    int64_t* need;
    uint8_t* flags;
    int64_t* beff_out;
    int32_t* q_out;
    uint32_t* dev_err;
};

// ---------------------------------------------------------------------------
// Every arrival against the reported state
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kIndNT) void static_independent(StaticArgs a) {
    __shared__ int64_t lb[kIndTile];
    __shared__ int32_t lq[kIndTile];
    const int64_t first = int64_t(blockIdx.x) * (kIndNT * kIndPer) + threadIdx.x;
    int64_t need[kIndPer];
    int32_t feas[kIndPer], most[kIndPer], fq[kIndPer];
    int64_t mb[kIndPer];
    bool bad = false;
#pragma unroll
    for (int k = 0; k < kIndPer; ++k) {
        const int64_t i = first + k * kIndNT;
        need[k] = -1;
        if (i < a.A && a.aU[i] >= 0) {
            const int32_t pr = a.ap[i];
            bad |= pr < 0;
            need[k] = ceil_blocks(int64_t(pr) + a.aU[i], a.S);
        }
        feas[k] = -1;
        fq[k] = 0;
        most[k] = -1;
        mb[k] = 0;
    }
    if (bad) raise_error(a.dev_err, MAPS_ERR_NEG_LEN);
    for (int32_t t0 = 0; t0 < a.D; t0 += kIndTile) {
        const int32_t n = a.D - t0 < kIndTile ? a.D - t0 : kIndTile;
        __syncthreads();
        for (int j = threadIdx.x; j < n; j += kIndNT) {
            lb[j] = a.beff[t0 + j];
            lq[j] = a.qlen[t0 + j];
        }
        __syncthreads();
        for (int j = 0; j < n; ++j) {
            const int64_t B = lb[j];
            const int32_t Q = lq[j];
            const int32_t d = t0 + j;
#pragma unroll
            for (int k = 0; k < kIndPer; ++k) {
                // ascending decoders: strict comparisons keep the lowest index on ties
                if (need[k] <= B && (feas[k] < 0 || Q < fq[k])) { feas[k] = d; fq[k] = Q; }
                if (most[k] < 0 || B > mb[k]) { most[k] = d; mb[k] = B; }
            }
        }
    }
    // the feasible decoder's B_eff for the flag: feasible means need <= B_eff
#pragma unroll
    for (int k = 0; k < kIndPer; ++k) {
        const int64_t i = first + k * kIndNT;
        if (i >= a.A) continue;
        int32_t d;
        uint8_t f;
        if (a.aU[i] < 0) {
            d = int32_t((a.rr_offset + i) % a.D);
            f = 2;
        } else if (a.policy == MAPS_POLICY_MQ && feas[k] >= 0) {
            d = feas[k];
            f = 1;
        } else {
            d = most[k];
            f = need[k] <= mb[k] ? 1 : 0;
        }
        a.choice[i] = d;
        a.need[i] = need[k];
        a.flags[i] = f;
    }
}

__global__ void static_copy_state(StaticArgs a) {
    for (int32_t d = blockIdx.x * blockDim.x + threadIdx.x; d < a.D; d += gridDim.x * blockDim.x) {
        if (a.beff_out) a.beff_out[d] = a.beff[d];
        if (a.q_out) a.q_out[d] = a.qlen[d];
    }
}

// ---------------------------------------------------------------------------
// One arrival after another, with reservation
// ---------------------------------------------------------------------------
// 64-bit wavefront minimum and maximum as two 32-bit reductions, high word
// first (a 32-bit DPP step is one instruction, a 64-bit one is five)
__device__ inline uint32_t wave_max_u32(uint32_t v) {
    return wave_last(wave_incl_scan(v, 0u, [](uint32_t x, uint32_t y) { return x > y ? x : y; }));
}

__device__ inline uint64_t wave_max_u64(uint64_t v) {
    const uint32_t hi = wave_max_u32(uint32_t(v >> 32));
    const uint32_t lo = wave_max_u32(uint32_t(v >> 32) == hi ? uint32_t(v) : 0u);
    return (uint64_t(hi) << 32) | lo;
}

__device__ inline uint64_t wave_min_u64(uint64_t v) {
    return ~wave_max_u64(~v);
}

// B_need of every arrival (-1 without a bound), in parallel before the chain
__global__ void static_need(StaticArgs a) {
    bool bad = false;
    for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < a.A; i += int64_t(gridDim.x) * blockDim.x) {
        const int32_t U = a.aU[i], p = a.ap[i];
        bad |= U >= 0 && p < 0;
        a.need[i] = U < 0 ? -1 : ceil_blocks(int64_t(p) + U, a.S);
    }
    if (bad) raise_error(a.dev_err, MAPS_ERR_NEG_LEN);
}

// Largest-B_eff key of one decoder: (B_eff + 2^52) above (1023 - decoder);
// 0 (below every key) for a slot past the last decoder.
__device__ inline uint64_t best_b_key(int64_t B, int32_t d, int32_t D) {
    return d < D ? (uint64_t(B + kBlockLimit) << 10) | uint64_t(1023 - d) : 0;
}

// The same order in 32 bits for a run of arrivals whose needs sum to less
// than 2^21 blocks: B_eff relative to the largest one at the run's start,
// `top` (B - top + 2^21, at least 1 for every B the largest can still reach,
// 0 for the lower ones, which cannot become the largest within the run).
constexpr int64_t kNarrowSpan = int64_t(1) << 21;
__device__ inline uint32_t best_b_key32(int64_t B, int64_t top, int32_t d, int32_t D) {
    if (d >= D) return 0;
    const int64_t r = B - top + kNarrowSpan;
    return (uint32_t(r > 0 ? r : 0) << 10) | uint32_t(1023 - d);
}

// kSlots decoders per lane: decoder lane + 64 s in slot s, with its B_eff,
// queue length and largest-B_eff key in registers.  The largest key over all
// decoders is kept between arrivals (only the chosen decoder's changes): an
// arrival whose B_need exceeds it takes that decoder at once; only a
// feasible shortest-queue choice scans every decoder.  The chosen decoder's
// lane and slot are the same in every lane, so its update is one scalar
// branch to one slot's code.  The arrivals go 64 at a time (one per lane,
// read out with readlane); a run of 64 whose needs sum to less than 2^21
// blocks and whose queues stay below 2^21 keeps its keys in 32 bits (one DPP
// reduction per arrival instead of two), any other run in 64 bits.
template <int kSlots, bool kNarrow>
__device__ __forceinline__ void reserve_run(const StaticArgs& a, int64_t c0, int cnt, int64_t my_need,
                                            int64_t (&B)[kSlots], int64_t (&Q)[kSlots], int64_t& bmax_all,
                                            bool& range_bad, int32_t& out_d, uint8_t& out_f) {
    using Key = typename std::conditional<kNarrow, uint32_t, uint64_t>::type;
    const int lane = threadIdx.x;
    const bool mq = a.policy == MAPS_POLICY_MQ;
    const int64_t top = bmax_all;   // the largest B_eff at the run's start
    Key K[kSlots];
    auto key_of = [&](int64_t b, int32_t d) -> Key {
        if constexpr (kNarrow) return best_b_key32(b, top, d, a.D);
        else return best_b_key(b, d, a.D);
    };
    auto wave_max = [&](Key v) -> Key {
        if constexpr (kNarrow) return wave_max_u32(v);
        else return wave_max_u64(v);
    };
    auto lane_best = [&]() {
        Key m = K[0];
#pragma unroll
        for (int s = 1; s < kSlots; ++s) m = K[s] > m ? K[s] : m;
        return m;
    };
#pragma unroll
    for (int s = 0; s < kSlots; ++s) K[s] = key_of(B[s], lane + s * kWave);
    Key kb = wave_max(lane_best());
    auto largest = [&](Key k) -> int64_t {
        if constexpr (kNarrow) return top + int64_t(k >> 10) - kNarrowSpan;
        else return int64_t(k >> 10) - kBlockLimit;
    };
    for (int j = 0; j < cnt; ++j) {
        const int64_t need = (int64_t(uint32_t(__builtin_amdgcn_readlane(int32_t(uint64_t(my_need) >> 32), j)))
                              << 32) |
                             uint32_t(__builtin_amdgcn_readlane(int32_t(my_need), j));
        int32_t best;
        uint8_t f;
        if (need < 0) {
            best = int32_t((a.rr_offset + c0 + j) % a.D);
            f = 2;
        } else {
            const int64_t bmax = largest(kb);
            if (mq && need <= bmax) {
                // feasible decoders exist: (Q, decoder) among them, smallest first
                Key kf = ~Key(0);
#pragma unroll
                for (int s = 0; s < kSlots; ++s) {
                    const int32_t d = lane + s * kWave;
                    const Key k1 = kNarrow ? Key((uint64_t(Q[s]) << 10) | uint64_t(d))
                                           : Key((uint64_t(Q[s]) << 20) | uint64_t(d));
                    if (d < a.D && need <= B[s] && k1 < kf) kf = k1;
                }
                kf = ~wave_max(~kf);
                best = int32_t(kf & (kNarrow ? 0x3FF : 0xFFFFF));
                f = 1;
            } else {
                best = 1023 - int32_t(kb & 1023);
                f = need <= bmax ? 1 : 0;
            }
        }
        // the owning lane reserves and enqueues; a reservation changes the largest B_eff
        const int owner = best % kWave, slot = best / kWave;
        if (lane == owner) {
#pragma unroll
            for (int s = 0; s < kSlots; ++s) {
                if (s == slot) {   // uniform: a scalar branch
                    if (need >= 0) {
                        B[s] -= need;
                        K[s] = key_of(B[s], best);
                    }
                    Q[s] += 1;
                    if constexpr (!kNarrow) range_bad |= B[s] <= -kBlockLimit || B[s] >= kBlockLimit;
                }
            }
        }
        if (need >= 0) kb = wave_max(lane_best());
        if (lane == j) {
            out_d = best;
            out_f = f;
        }
    }
    bmax_all = largest(kb);
    if constexpr (kNarrow) {
        // B only decreases: the run's end shows whether any left the packed-key range
#pragma unroll
        for (int s = 0; s < kSlots; ++s) range_bad |= B[s] <= -kBlockLimit;
    }
}

template <int kSlots>
__global__ __launch_bounds__(kWave) void static_reserve(StaticArgs a) {
    const int lane = threadIdx.x;
    int64_t B[kSlots];
    int64_t Q[kSlots];
    uint64_t k0 = 0;
#pragma unroll
    for (int s = 0; s < kSlots; ++s) {
        const int32_t d = lane + s * kWave;
        B[s] = d < a.D ? a.beff[d] : 0;
        Q[s] = d < a.D ? a.qlen[d] : 0;
        const uint64_t k = best_b_key(B[s], d, a.D);
        k0 = k > k0 ? k : k0;
    }
    int64_t bmax_all = int64_t(wave_max_u64(k0) >> 10) - kBlockLimit;   // the largest B_eff
    bool range_bad = false;
    for (int64_t c0 = 0; c0 < a.A; c0 += kWave) {
        const int64_t mine = c0 + lane;
        const int64_t my_need = mine < a.A ? a.need[mine] : -1;
        int32_t out_d = 0;
        uint8_t out_f = 0;
        const int cnt = a.A - c0 < kWave ? int(a.A - c0) : kWave;
        // the run's needs and the longest queue after it decide the key width (the same in every lane)
        int64_t qmax = 0;
#pragma unroll
        for (int s = 0; s < kSlots; ++s) qmax = Q[s] > qmax ? Q[s] : qmax;
        qmax = int64_t(wave_max_u64(uint64_t(qmax)));
        const int64_t need_sum = wave_reduce_add(my_need > 0 ? my_need : int64_t(0));
        if (need_sum < kNarrowSpan - 1 && qmax + kWave < kNarrowSpan)
            reserve_run<kSlots, true>(a, c0, cnt, my_need, B, Q, bmax_all, range_bad, out_d, out_f);
        else
            reserve_run<kSlots, false>(a, c0, cnt, my_need, B, Q, bmax_all, range_bad, out_d, out_f);
        if (mine < a.A) {
            a.choice[mine] = out_d;
            a.flags[mine] = out_f;
        }
    }
#pragma unroll
    for (int s = 0; s < kSlots; ++s) {
        const int32_t d = lane + s * kWave;
        if (d < a.D) {
            if (a.beff_out) a.beff_out[d] = B[s];
            if (a.q_out) a.q_out[d] = int32_t(Q[s]);
        }
    }
    if (range_bad) raise_error(a.dev_err, MAPS_ERR_BLOCK_RANGE);
}

// every initial B_eff inside the packed-key range
__global__ void static_check_range(StaticArgs a) {
    bool bad = false;
    for (int32_t d = blockIdx.x * blockDim.x + threadIdx.x; d < a.D; d += gridDim.x * blockDim.x)
        bad |= a.beff[d] <= -kBlockLimit || a.beff[d] >= kBlockLimit;
    if (bad) raise_error(a.dev_err, MAPS_ERR_BLOCK_RANGE);
}

}  // namespace
}  // namespace maps

using namespace maps;

extern "C" maps_status maps_rsc_state(int32_t D, const int64_t* seg_off, int64_t n_total, const int32_t* prompt,
                                      const int32_t* generated, const int32_t* upper, const uint8_t* in_flight,
                                      const int32_t* capacity,
                                      int32_t block_size, int64_t* b_free, int64_t* b_res, int64_t* b_eff,
                                      uint32_t* dev_err, hipStream_t stream) {
    if (D < 1 || n_total < 0 || block_size < 1) return MAPS_E_SIZE;
    if (!seg_off || !capacity || !b_free || !b_res || !b_eff || !dev_err ||
        (n_total > 0 && (!prompt || !generated || !upper)))
        return MAPS_E_NULL;
    hipLaunchKernelGGL(rsc_state, dim3(unsigned(D)), dim3(kRscNT), 0, stream, D, seg_off, n_total, prompt,
                       generated, upper, in_flight, capacity, block_size, b_free, b_res, b_eff, dev_err);
    MAPS_CHECK_LAUNCH();
    return MAPS_OK;
}

extern "C" maps_status maps_place_static(int32_t D, const int64_t* b_eff, const int32_t* queue_len,
                                         int32_t block_size, const int32_t* a_prompt, const int32_t* a_upper,
                                         int64_t A, int32_t policy, int64_t rr_offset, int32_t reserve,
                                         int32_t* choice, int64_t* b_need, uint8_t* flags, int64_t* b_eff_out,
                                         int32_t* queue_out, uint32_t* dev_err, hipStream_t stream) {
    if (D < 1 || A < 0 || block_size < 1 || rr_offset < 0 || (reserve && D > MAPS_MAX_RESERVE_DECODERS))
        return MAPS_E_SIZE;
    if (policy != MAPS_POLICY_MQ && policy != MAPS_POLICY_MC) return MAPS_E_POLICY;
    if (!b_eff || !queue_len || !dev_err || (A > 0 && (!a_prompt || !a_upper || !choice || !b_need || !flags)))
        return MAPS_E_NULL;
    StaticArgs a{D, b_eff, queue_len, block_size, a_prompt, a_upper, A, policy, rr_offset, choice, b_need, flags,
                 b_eff_out, queue_out, dev_err};
    if (reserve) {
        hipLaunchKernelGGL(static_check_range, dim3(unsigned((D + 255) / 256)), dim3(256), 0, stream, a);
        MAPS_CHECK_LAUNCH();
        if (A > 0) {
            const int64_t nblk = (A + 255) / 256;
            hipLaunchKernelGGL(static_need, dim3(unsigned(nblk < 4096 ? nblk : 4096)), dim3(256), 0, stream, a);
            MAPS_CHECK_LAUNCH();
        }
        const int slots = (D + kWave - 1) / kWave;
        if (slots <= 1) hipLaunchKernelGGL(static_reserve<1>, dim3(1), dim3(kWave), 0, stream, a);
        else if (slots <= 2) hipLaunchKernelGGL(static_reserve<2>, dim3(1), dim3(kWave), 0, stream, a);
        else if (slots <= 4) hipLaunchKernelGGL(static_reserve<4>, dim3(1), dim3(kWave), 0, stream, a);
        else if (slots <= 8) hipLaunchKernelGGL(static_reserve<8>, dim3(1), dim3(kWave), 0, stream, a);
        else hipLaunchKernelGGL(static_reserve<kResSlots>, dim3(1), dim3(kWave), 0, stream, a);
        MAPS_CHECK_LAUNCH();
        return MAPS_OK;
    }
    if (A > 0) {
        const int64_t blocks = (A + kIndNT * kIndPer - 1) / (kIndNT * kIndPer);
        hipLaunchKernelGGL(static_independent, dim3(unsigned(blocks)), dim3(kIndNT), 0, stream, a);
        MAPS_CHECK_LAUNCH();
    }
    if (b_eff_out || queue_out) {
        hipLaunchKernelGGL(static_copy_state, dim3(unsigned((D + 255) / 256)), dim3(256), 0, stream, a);
        MAPS_CHECK_LAUNCH();
    }
    return MAPS_OK;
}
