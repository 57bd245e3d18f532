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

// One thread per (sequence, row i, column j): j is on i's root path iff
// walking up from i (pruned indices decrease towards the root) meets j.
__global__ void k_tree_mask(TreeDev t, int R, uint8_t* mask, int32_t* depth) {
    const int n = R + 1;
    const int64_t total = (int64_t)t.B * n * n;
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int b = (int)(e / ((int64_t)n * n));
        const int i = (int)((e / n) % n);
        const int j = (int)(e % n);
        const int64_t nb = (int64_t)b * t.NN;
        int p = i;
        // at most depth (<= 15) steps; p > j >= 0 keeps the root's parent unread
        for (int s = 0; s < 16 && p > j; ++s) p = t.pidx[nb + t.par[nb + t.porder[nb + p]]];
        if (mask) mask[e] = (p == j) ? 1 : 0;
        if (depth && j == 0) depth[(int64_t)b * n + i] = t.meta[nb + t.porder[nb + i]] & 0xFF;
    }
}

hipError_t launch_tree_mask(const TreeDev& t, int R, uint8_t* mask, int32_t* depth,
                            hipStream_t s) {
    const int64_t n = (int64_t)t.B * (R + 1) * (R + 1);
    const int blocks = (int)((n + 255) / 256 < 8192 ? (n + 255) / 256 : 8192);
    k_tree_mask<<<blocks, 256, 0, s>>>(t, R, mask, depth);
    return hipGetLastError();
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
