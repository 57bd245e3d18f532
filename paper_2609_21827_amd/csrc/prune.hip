// Global pruning of the draft tree (App. C.1, "Path scores and global
// pruning" and "Tie-breaking rule"): keep the R non-root nodes with the
// highest path score, ties by depth (shallower first), then left-to-right
// sibling order.  Scores never grow along a path (Lemma 2) and the tie-break
// ranks a parent before its children, so the kept set is ancestor-closed.
//
// One block per sequence orders all nodes by their 128-bit priority key
// (keys are unique): a bitonic sort in LDS, or, for trees too large for it,
// a counting rank (each node's rank is the number of larger keys).
#include "rheo_device.h"
#include "rheo_state.h"

namespace rheo {

constexpr int NTR = 256;
constexpr int SORT_MAX = 2048;   // nodes the bitonic sort holds in LDS

__device__ __forceinline__ bool key_gt(const ulonglong2& a, const ulonglong2& b) {
    return a.x > b.x || (a.x == b.x && a.y > b.y);
}

__global__ __launch_bounds__(NTR) void k_prune(TreeDev t, int R) {
    extern __shared__ ulonglong2 s_dyn[];
    const int b = blockIdx.x;
    const int tid = threadIdx.x;
    const int n = t.NN - 1;               // non-root nodes, uids 1..NN-1
    const int64_t nb = (int64_t)b * t.NN;
    if (tid == 0) {
        t.pidx[nb] = 0;
        t.porder[nb] = 0;
    }
    if (n <= SORT_MAX) {
        int N = 1;
        while (N < n) N <<= 1;
        ulonglong2* s_key = s_dyn;
        uint16_t* s_idx = (uint16_t*)(s_dyn + N);
        for (int i = tid; i < N; i += NTR) {
            if (i < n) {
                const int64_t o = nb + 1 + i;
                uint64_t hi, lo;
                prio_key(t.score[o], t.meta[o] & 0xFF, t.path[o], hi, lo);
                s_key[i] = make_ulonglong2(hi, lo);
            } else {
                s_key[i] = make_ulonglong2(0ull, 0ull);   // below every node
            }
            s_idx[i] = (uint16_t)i;
        }
        __syncthreads();
        // descending bitonic sort of N keys (N / 2 compare-exchanges a stage)
        for (int k = 2; k <= N; k <<= 1) {
            for (int j = k >> 1; j > 0; j >>= 1) {
                for (int p = tid; p < N / 2; p += NTR) {
                    const int i = 2 * p - (p & (j - 1));      // lower index of the pair
                    const int l = i + j;
                    const bool desc = (i & k) == 0;
                    const ulonglong2 x = s_key[i], y = s_key[l];
                    if (key_gt(y, x) == desc) {
                        s_key[i] = y;
                        s_key[l] = x;
                        const uint16_t ti = s_idx[i];
                        s_idx[i] = s_idx[l];
                        s_idx[l] = ti;
                    }
                }
                __syncthreads();
            }
        }
        for (int r = tid; r < n; r += NTR) {
            const int i = s_idx[r];
            if (r < R) {
                t.pidx[nb + 1 + i] = r + 1;
                t.porder[nb + r + 1] = 1 + i;
            } else {
                t.pidx[nb + 1 + i] = -1;
            }
        }
    } else {
        ulonglong2* s_key = s_dyn;
        int16_t* s_rank = (int16_t*)(s_dyn + n);
        for (int i = tid; i < n; i += NTR) {
            const int64_t o = nb + 1 + i;
            uint64_t hi, lo;
            prio_key(t.score[o], t.meta[o] & 0xFF, t.path[o], hi, lo);
            s_key[i] = make_ulonglong2(hi, lo);
        }
        __syncthreads();
        rank_keys128<NTR>(s_key, n, s_rank);
        __syncthreads();
        for (int i = tid; i < n; i += NTR) {
            const int rk = s_rank[i];
            if (rk < R) {
                t.pidx[nb + 1 + i] = rk + 1;
                t.porder[nb + rk + 1] = 1 + i;
            } else {
                t.pidx[nb + 1 + i] = -1;
            }
        }
    }
    __syncthreads();
    // ancestor closure (a violated invariant raises the sticky error flag)
    for (int i = tid; i < n; i += NTR) {
        const int64_t o = nb + 1 + i;
        if (t.pidx[o] > 0 && t.pidx[nb + t.par[o]] < 0) atomicOr(t.err, 2);
    }
}

hipError_t launch_prune(const TreeDev& t, int R, hipStream_t s) {
    const int n = t.NN - 1;
    int N = 1;
    while (N < n) N <<= 1;
    const size_t shm = n <= SORT_MAX
        ? (sizeof(ulonglong2) + sizeof(uint16_t)) * (size_t)N + 16
        : (sizeof(ulonglong2) + sizeof(int16_t)) * (size_t)n + 16;
    k_prune<<<t.B, NTR, shm, s>>>(t, R);
    return hipGetLastError();
}

}  // namespace rheo
