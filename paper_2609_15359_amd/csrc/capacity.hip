// KV capacity in bytes to tokens (App. A: KV tokens and bytes are related by
// model constants): tokens[d] = floor(bytes[d] / bytes_per_token).
#include "maps_internal.hpp"

namespace maps {
namespace {

__global__ __launch_bounds__(256) void capacity_tokens_kernel(const int64_t* __restrict__ bytes, int32_t D,
                                                              int64_t per_token, int32_t* __restrict__ tokens,
                                                              uint32_t* dev_err) {
    bool neg = false, range = false;
    for (int32_t d = int32_t(blockIdx.x) * 256 + int32_t(threadIdx.x); d < D; d += int32_t(gridDim.x) * 256) {
        const int64_t b = bytes[d];
        int64_t t = b < 0 ? 0 : b / per_token;   // floor: b >= 0 here
        neg |= b < 0;
        if (t > INT32_MAX) { range = true; t = INT32_MAX; }
        tokens[d] = int32_t(t);
    }
    if (neg) raise_error(dev_err, MAPS_ERR_NEG_LEN);
    if (range) raise_error(dev_err, MAPS_ERR_INT32_RANGE);
}

}  // namespace
}  // namespace maps

using namespace maps;

extern "C" maps_status maps_capacity_tokens(const int64_t* capacity_bytes, int32_t D, int64_t bytes_per_token,
                                            int32_t* capacity_tokens, uint32_t* dev_err, hipStream_t stream) {
    if (D < 1 || bytes_per_token < 1) return MAPS_E_SIZE;
    if (!capacity_bytes || !capacity_tokens || !dev_err) return MAPS_E_NULL;
    const int32_t blocks = (D + 255) / 256 < 1024 ? (D + 255) / 256 : 1024;
    hipLaunchKernelGGL(capacity_tokens_kernel, dim3(blocks), dim3(256), 0, stream, capacity_bytes, D,
                       bytes_per_token, capacity_tokens, dev_err);
    MAPS_CHECK_LAUNCH();
    return MAPS_OK;
}
