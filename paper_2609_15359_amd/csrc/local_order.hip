// Local SJF order and admission (Sec. 3.3, Eq. (7); App. A, Eq. (10)): the
// launch of maps_local_order (one workgroup per decoder; the device code is
// in order_core.hpp).
#include "order_core.hpp"

namespace maps {
namespace {

__global__ __launch_bounds__(order::kOrderNT) void local_order_kernel(order::LocalArgs g) {
    order::order_queue(g, int32_t(blockIdx.x));
}

}  // namespace
}  // namespace maps

using namespace maps;

extern "C" size_t maps_local_order_workspace_size(int32_t, int64_t) { return 0; }

extern "C" maps_status maps_local_order(const void* snapshot, int32_t D, int32_t u_max, const int32_t* capacity,
                                        const int64_t* q_off, int64_t total, const int32_t* q_prompt,
                                        const int32_t* q_upper, const int32_t* q_wait_ms, int32_t max_wait_ms,
                                        int32_t* order, int32_t* admitted, uint32_t* dev_err, void* workspace,
                                        size_t workspace_bytes, hipStream_t stream) {
    (void)workspace;
    (void)workspace_bytes;
    if (D < 1 || total < 0 || u_max < 0 || u_max > MAPS_MAX_U_MAX) return MAPS_E_SIZE;
    if (!snapshot || !capacity || !q_off || !admitted || !dev_err ||
        (total > 0 && (!q_prompt || !q_upper || !order)))
        return MAPS_E_NULL;
    order::LocalArgs a;
    a.L = snap_layout(D, 0, u_max);
    a.snap = snapshot;
    a.cap = capacity;
    a.q_off = q_off;
    a.total = total;
    a.qp = q_prompt;
    a.qU = q_upper;
    a.qwait = q_wait_ms;
    a.max_wait = max_wait_ms;
    a.order = order;
    a.admitted = admitted;
    a.dev_err = dev_err;
    hipLaunchKernelGGL(local_order_kernel, dim3(D), dim3(order::kOrderNT), 0, stream, a);
    MAPS_CHECK_LAUNCH();
    return MAPS_OK;
}

extern "C" const char* maps_status_string(maps_status status) {
    switch (status) {
        case MAPS_OK: return "ok";
        case MAPS_E_NULL: return "a required pointer is NULL";
        case MAPS_E_SIZE: return "a count or size is out of range";
        case MAPS_E_ALPHA: return "alpha_ppm is not in (0, 1000000)";
        case MAPS_E_WORKSPACE: return "workspace smaller than the size query";
        case MAPS_E_HIP: return "HIP runtime error";
        case MAPS_E_POLICY: return "unknown placement policy";
        case MAPS_E_BUFFER: return "snapshot buffer smaller than maps_snapshot_bytes()";
        default: return "unknown status";
    }
}
