// Global pruning of the draft tree (App. C.1, "Path scores and global
// pruning" and "Tie-breaking rule"): keep the R non-root nodes with the
// highest path score, ties by depth (shallower first), then left-to-right
// sibling order.  Scores never grow along a path (Lemma 2) and the tie-break
// ranks a parent before its children, so the kept set is ancestor-closed.
//
// PSPLIT blocks per sequence each load all of its nodes' 128-bit priority
// keys (unique) into LDS and rank their share of the nodes by counting the
// larger keys, several lanes per node.  Every block also checks, for its
// nodes, that a parent's key is larger than its child's: that is what makes
// the kept set ancestor-closed, checked without waiting for other blocks.
#include "rheo_device.h"
#include "rheo_state.h"

namespace rheo {

constexpr int NTR = 256;
constexpr int PSPLIT = 16;         // blocks per sequence

__global__ __launch_bounds__(NTR) void k_prune(TreeDev t, int R) {
    extern __shared__ ulonglong2 s_key[];    // the sequence's n keys
    const int b = blockIdx.x / PSPLIT, part = blockIdx.x % PSPLIT;
    const int tid = threadIdx.x;
    const int n = t.NN - 1;               // non-root nodes, uids 1..NN-1
    const int64_t nb = (int64_t)b * t.NN;
    if (part == 0 && tid == 0) {
        t.pidx[nb] = 0;
        t.porder[nb] = 0;
    }
    for (int i = tid; i < n; i += NTR) {
        const int64_t o = nb + 1 + i;
        uint64_t hi, lo;
        prio_key(t.score[o], t.meta[o] & 0xFF, t.path[o], hi, lo);
        s_key[i] = make_ulonglong2(hi, lo);
    }
    __syncthreads();
    // this block's nodes [i0, i1), F lanes per node, each over every F-th key
    const int per = (n + PSPLIT - 1) / PSPLIT;
    const int i0 = min(n, part * per), i1 = min(n, i0 + per);
    const int m = i1 - i0;
    int F = 1;
    while (F < 16 && 2 * F * m <= NTR) F *= 2;
    const int sub = tid % F;
    for (int base = 0; base < m; base += NTR / F) {
        const int i = i0 + base + tid / F;
        int cnt = 0;
        ulonglong2 k = make_ulonglong2(~0ull, ~0ull);
        if (i < i1) k = s_key[i];
#pragma unroll 8
        for (int j = sub; j < n; j += F) {
            const ulonglong2 x = s_key[j];
            cnt += (int)(x.x > k.x) | ((int)(x.x == k.x) & (int)(x.y > k.y));
        }
        for (int o = 1; o < F; o <<= 1) cnt += __shfl_xor(cnt, o);
        if (i < i1 && sub == 0) {
            const int64_t o = nb + 1 + i;
            if (cnt < R) {
                t.pidx[o] = cnt + 1;
                t.porder[nb + cnt + 1] = 1 + i;
            } else {
                t.pidx[o] = -1;
            }
            // a parent outranks its child (raises the sticky error flag if not)
            const int p = t.par[o];
            if (p > 0) {
                const ulonglong2 pk = s_key[p - 1];
                if (!(pk.x > k.x || (pk.x == k.x && pk.y > k.y))) atomicOr(t.err, 2);
            }
        }
    }
}

hipError_t launch_prune(const TreeDev& t, int R, hipStream_t s) {
    const int n = t.NN - 1;
    k_prune<<<t.B * PSPLIT, NTR, sizeof(ulonglong2) * (size_t)n, s>>>(t, R);
    return hipGetLastError();
}

}  // namespace rheo
