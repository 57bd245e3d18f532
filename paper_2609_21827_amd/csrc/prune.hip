// Global pruning of the draft tree (App. C.1, "Path scores and global
// pruning" and "Tie-breaking rule"): keep the R non-root nodes with the
// highest path score, ties by depth (shallower first), then left-to-right
// sibling order.  Scores never grow along a path (Lemma 2) and the tie-break
// ranks a parent before its children, so the kept set is ancestor-closed.
//
// One block per sequence ranks all nodes by counting (each node's rank is
// the number of nodes with a larger 128-bit priority key; keys are unique),
// several lanes sharing each node's comparisons.
#include "rheo_device.h"
#include "rheo_state.h"

namespace rheo {

template <int NT>
__global__ __launch_bounds__(NT) void k_prune(TreeDev t, int R) {
    extern __shared__ uint64_t s_dyn[];
    const int b = blockIdx.x;
    const int n = t.NN - 1;               // non-root nodes, uids 1..NN-1
    uint64_t* s_hi = s_dyn;
    uint64_t* s_lo = s_dyn + n;
    const int64_t nb = (int64_t)b * t.NN;
    for (int i = threadIdx.x; i < n; i += NT) {
        const int64_t o = nb + 1 + i;
        uint64_t hi, lo;
        prio_key(t.score[o], t.meta[o] & 0xFF, t.path[o], hi, lo);
        s_hi[i] = hi;
        s_lo[i] = lo;
    }
    if (threadIdx.x == 0) {
        t.pidx[nb] = 0;
        t.porder[nb] = 0;
    }
    __syncthreads();
    int16_t* s_rank = (int16_t*)(s_dyn + 2 * n);
    rank_keys128<NT>(s_hi, s_lo, n, s_rank);
    __syncthreads();
    for (int i = threadIdx.x; i < n; i += NT) {
        const int rk = s_rank[i];
        if (rk < R) {
            t.pidx[nb + 1 + i] = rk + 1;
            t.porder[nb + rk + 1] = 1 + i;
        } else {
            t.pidx[nb + 1 + i] = -1;
        }
    }
    __syncthreads();
    // ancestor closure (a violated invariant raises the sticky error flag)
    for (int i = threadIdx.x; i < n; i += NT) {
        const int64_t o = nb + 1 + i;
        if (t.pidx[o] > 0 && t.pidx[nb + t.par[o]] < 0) atomicOr(t.err, 2);
    }
}

hipError_t launch_prune(const TreeDev& t, int R, hipStream_t s) {
    const size_t shm = (2 * sizeof(uint64_t) + sizeof(int16_t)) * (size_t)(t.NN - 1) + 16;
    k_prune<1024><<<t.B, 1024, shm, s>>>(t, R);
    return hipGetLastError();
}

}  // namespace rheo
