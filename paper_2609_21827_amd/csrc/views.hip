// Small copy-out kernels for the ABI's view calls.
#include "rheo_device.h"
#include "rheo_state.h"

namespace rheo {

__global__ void k_read_nodes(TreeDev t, int32_t* token, int32_t* parent, int32_t* depth,
                             int32_t* slot, int32_t* kind, double* proxy, double* qtrue,
                             double* score) {
    const int64_t n = (int64_t)t.B * t.NN;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int meta = t.meta[i];
        if (token) token[i] = t.tok[i];
        if (parent) parent[i] = t.par[i];
        if (depth) depth[i] = meta & 0xFF;
        if (slot) slot[i] = (meta >> 8) & 0xFF;
        if (kind) kind[i] = (meta >> 16) & 0xFF;
        if (proxy) proxy[i] = t.proxy[i];
        if (qtrue) qtrue[i] = t.qtrue[i];
        if (score) score[i] = t.score[i];
    }
}

__global__ void k_pruned_view(TreeDev t, int R, int32_t* parent, int32_t* token) {
    const int64_t n = (int64_t)t.B * (R + 1);
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int b = (int)(i / (R + 1));
        const int k = (int)(i % (R + 1));
        const int64_t nb = (int64_t)b * t.NN;
        const int uid = t.porder[nb + k];
        if (parent) parent[i] = (k == 0) ? -1 : t.pidx[nb + t.par[nb + uid]];
        if (token) token[i] = (k == 0) ? -1 : t.tok[nb + uid];
    }
}

hipError_t launch_read_nodes(const TreeDev& t, int32_t* token, int32_t* parent,
                             int32_t* depth, int32_t* slot, int32_t* kind, double* proxy,
                             double* qtrue, double* score, hipStream_t s) {
    const int64_t n = (int64_t)t.B * t.NN;
    const int blocks = (int)((n + 255) / 256 < 4096 ? (n + 255) / 256 : 4096);
    k_read_nodes<<<blocks, 256, 0, s>>>(t, token, parent, depth, slot, kind, proxy, qtrue,
                                        score);
    return hipGetLastError();
}

hipError_t launch_pruned_view(const TreeDev& t, int R, int32_t* parent, int32_t* token,
                              hipStream_t s) {
    const int64_t n = (int64_t)t.B * (R + 1);
    const int blocks = (int)((n + 255) / 256 < 4096 ? (n + 255) / 256 : 4096);
    k_pruned_view<<<blocks, 256, 0, s>>>(t, R, parent, token);
    return hipGetLastError();
}

}  // namespace rheo
