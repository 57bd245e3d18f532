// Device helpers shared by the sparse and dense pool kernels: ranking by
// counting, sums over the threads forming a pool, a child record, and the
// frontier selection of a sequence.
#pragma once

#include "rheo_device.h"
#include "rheo_state.h"

namespace rheo {

// Ranks of two keys at once (counts of larger keys among n unique keys in
// LDS, 16-byte aligned); 16 keys per step keep eight loads in flight.
__device__ __forceinline__ void count_greater2(const uint64_t* keys, int n, uint64_t k0,
                                               uint64_t k1, int& c0, int& c1) {
    const ulonglong2* kp = (const ulonglong2*)keys;
    int a0 = 0, a1 = 0;
    const int np = n >> 1;
#pragma unroll 8
    for (int j = 0; j < np; ++j) {
        const ulonglong2 x = kp[j];
        a0 += (int)(x.x > k0) + (int)(x.y > k0);
        a1 += (int)(x.x > k1) + (int)(x.y > k1);
    }
    if (n & 1) {
        const uint64_t x = keys[n - 1];
        a0 += (int)(x > k0);
        a1 += (int)(x > k1);
    }
    c0 = a0;
    c1 = a1;
}
// Ranks (counts of larger keys) of the n unique keys in LDS (16-byte
// aligned) by NT threads.  When the threads outnumber the keys, F adjacent
// lanes share a key (F a power of two, F * n <= NT, F <= 16), each counting
// over every F-th pair of keys, and their counts are added across the
// lanes; otherwise every thread ranks two keys at a time.
template <int NT>
__device__ __forceinline__ void rank_all(const uint64_t* keys, int n, int16_t* rank) {
    const int t = threadIdx.x % NT;
    int F = 1;
    while (F < 16 && 2 * F * n <= NT) F *= 2;
    if (F == 1) {
        for (int i = t; i < n; i += 2 * NT) {
            const int i2 = i + NT;
            int c0, c1;
            count_greater2(keys, n, keys[i], i2 < n ? keys[i2] : ~0ull, c0, c1);
            rank[i] = (int16_t)c0;
            if (i2 < n) rank[i2] = (int16_t)c1;
        }
        return;
    }
    const ulonglong2* kp = (const ulonglong2*)keys;
    const int i = t / F, sub = t % F;
    const uint64_t k = keys[i < n ? i : 0];
    const int np = n >> 1;
    int c = 0;
#pragma unroll 4
    for (int j = sub; j < np; j += F) {
        const ulonglong2 x = kp[j];
        c += (int)(x.x > k) + (int)(x.y > k);
    }
    if ((n & 1) && sub == 0) c += (int)(keys[n - 1] > k);
    for (int o = 1; o < F; o <<= 1) c += __shfl_xor(c, o);
    if (i < n && sub == 0) rank[i] = (int16_t)c;
}

// Synchronisation and sums over the NT threads that form a pool: one wave
// (small supports) or the whole block.
template <int NT>
__device__ __forceinline__ void psync() {
    if (NT == WAVE) wave_sync();
    else __syncthreads();
}

// Descending bitonic sort of n 64-bit keys in LDS (n a power of two) by NT
// threads; the caller has synchronised after writing the keys, and the sort
// ends with a barrier.  Compare-exchange pair i of a stage with distance j
// joins positions lo = ((i & ~(j - 1)) << 1) | (i & (j - 1)) and lo + j;
// for j <= WAVE every position a wave touches lies in the 2 * WAVE-wide
// window of its own pair indices, so consecutive such stages only need the
// wave's own accesses ordered.
template <int NT>
__device__ __forceinline__ void bitonic_sort_desc(uint64_t* k, int n) {
    const int tid = threadIdx.x % NT;
    const int half = n >> 1;
    for (int kk = 2; kk <= n; kk <<= 1) {
        for (int j = kk >> 1; j > 0; j >>= 1) {
            for (int i = tid; i < half; i += NT) {
                const int lo = ((i & ~(j - 1)) << 1) | (i & (j - 1));
                const int hi = lo + j;
                const uint64_t x = k[lo], y = k[hi];
                const bool desc = (lo & kk) == 0;
                if ((x < y) == desc) {
                    k[lo] = y;
                    k[hi] = x;
                }
            }
            const int jn = (j > 1) ? (j >> 1) : kk;      // the next stage's distance
            if (j > WAVE || jn > WAVE) psync<NT>();
            else wave_sync();
        }
    }
    psync<NT>();
}
template <int NT>
__device__ __forceinline__ uint64_t psum(uint64_t v, uint64_t* sh) {
    if (NT == WAVE) return wave_sum_u64(v);
    return block_sum_u64<NT>(v, sh);
}
template <int NT>
__device__ __forceinline__ void psum2(uint64_t a, uint64_t b, uint64_t* sh, uint64_t* ra,
                                      uint64_t* rb) {
    if (NT == WAVE) {
        *ra = wave_sum_u64(a);
        *rb = wave_sum_u64(b);
    } else {
        block_sum2_u64<NT>(a, b, sh, ra, rb);
    }
}
// Totals of a and b over the pool's NT threads and the exclusive prefix of
// b in thread order, in one exchange (sh: 2 * NT / WAVE words for a block).
template <int NT>
__device__ __forceinline__ void psum2_scan(uint64_t a, uint64_t b, uint64_t* sh, uint64_t* ra,
                                           uint64_t* rb, uint64_t* b_before) {
    const uint64_t binc = wave_incl_scan_u64(b);
    const uint64_t asum = wave_sum_u64(a);
    if (NT == WAVE) {
        *ra = asum;
        *rb = lane_u64(binc, WAVE - 1);
        *b_before = binc - b;
        return;
    }
    constexpr int NW = NT / WAVE;
    const int w = threadIdx.x / WAVE, l = threadIdx.x % WAVE;
    __syncthreads();
    if (l == WAVE - 1) {
        sh[w] = asum;
        sh[NW + w] = binc;
    }
    __syncthreads();
    uint64_t x = 0, y = 0, before = 0;
#pragma unroll
    for (int i = 0; i < NW; ++i) {
        x += sh[i];
        y += sh[NW + i];
        before += (i < w) ? sh[NW + i] : 0ull;
    }
    *ra = x;
    *rb = y;
    *b_before = before + binc - b;
}
// Exclusive prefix sum of one 64-bit value per thread over the pool's NT
// threads (sh: NT / WAVE words for a block); *total receives the sum.
template <int NT>
__device__ __forceinline__ uint64_t pscan_excl(uint64_t v, uint64_t* sh, uint64_t* total) {
    if (NT == WAVE) {
        const uint64_t inc = wave_incl_scan_u64(v);
        *total = lane_u64(inc, WAVE - 1);
        return inc - v;
    }
    return block_excl_scan_u64<NT>(v, sh, total);
}
template <int NT>
__device__ __forceinline__ bool pany(bool p) {
    if (NT == WAVE) return __ballot(p) != 0ull;
    return __syncthreads_or(p) != 0;
}

// The parent's path score and slot path (1 and 0 for the root), read early
// by the threads that later write the children.
struct ParentRec {
    double score;
    uint64_t path;
};
__device__ __forceinline__ ParentRec parent_rec(const TreeDev& t, int level, int64_t nb, int pu) {
    ParentRec p{1.0, 0ull};
    if (level > 0) {
        p.score = t.score[nb + pu];
        p.path = t.path[nb + pu];
    }
    return p;
}

// One child record of expanded row j (slot s, 0-based; App. C.1): the
// fields the frontier selection reads in other blocks (token, score, path)
// are published with agent-scope atomics.
// tail: the child's place in its parent's stored tail (-1: not in it)
__device__ __forceinline__ void emit_child(const TreeDev& t, int level, int64_t nb, int pu,
                                           const ParentRec& pr, int uid, int s, int kind,
                                           int tok, double proxy, double qtrue, int tail) {
    const double pscore = pr.score;
    const uint64_t ppath = pr.path;
    const int64_t o = nb + uid;
    t.par[o] = pu;
    t.tidx[o] = tail;
    t.meta[o] = (level + 1) | ((s + 1) << 8) | (kind << 16);
    t.proxy[o] = proxy;
    t.qtrue[o] = qtrue;
    t.first_child[o] = -1;
    t.exp_of[o] = -1;
    __hip_atomic_store(&t.tok[o], tok, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store((uint64_t*)&t.score[o], (uint64_t)__double_as_longlong(__dmul_rn(pscore, proxy)),
                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&t.path[o], ppath | ((uint64_t)(s + 1) << (56 - 4 * level)),
                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The root record (level 0 only).
__device__ __forceinline__ void emit_root(const TreeDev& t, int64_t nb) {
    t.tok[nb] = -1;
    t.par[nb] = -1;
    t.meta[nb] = 0;
    t.proxy[nb] = 1.0;
    t.qtrue[nb] = 1.0;
    t.score[nb] = 1.0;
    t.path[nb] = 0;
}

// The next frontier (Sec. 2.1; App. C.4, step 1: the next level expands the
// best-scoring new nodes).  Called by every block of the pool kernel once
// its children are written: the last row of sequence b to get here ranks
// the level's P * K new children by priority and keeps the best n_expand
// (the next level's rows take the Philox draw of each kept node's sampled
// slot themselves, keyed by this launch's rng_key).  s_hi and s_lo are
// LDS arrays of at least 256 entries the caller no longer needs.
__device__ __forceinline__ void select_frontier(const TreeDev& t, const LevelArgs& a, int b,
                                                uint64_t* s_hi, uint64_t* s_lo) {
    __shared__ int s_lastseq;
    const int tid = threadIdx.x;
    const int level = a.level;
    const int K = t.K, NE = t.NE;
    const int64_t nb = (int64_t)b * t.NN;
    if (level + 1 >= t.D) return;
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (tid == 0) {
        const uint32_t old = __hip_atomic_fetch_add(&t.seq_cnt[b], 1u, __ATOMIC_RELAXED,
                                                    __HIP_MEMORY_SCOPE_AGENT);
        s_lastseq = old == (uint32_t)(a.P - 1);
        if (s_lastseq) __hip_atomic_store(&t.seq_cnt[b], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();
    if (!s_lastseq) return;
    const int n = a.P * K;                       // <= 225
    const int cb = (level == 0) ? 1 : 1 + K + (level - 1) * NE * K;
    // every child's priority key and token in one round of loads
    int tok = -1;
    if (tid < n) {
        const int64_t o = nb + cb + tid;
        const double sc = __longlong_as_double((long long)__hip_atomic_load(
            (uint64_t*)&t.score[o], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
        const uint64_t pa = __hip_atomic_load(&t.path[o], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        tok = __hip_atomic_load(&t.tok[o], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        uint64_t hi, lo;
        prio_key(sc, level + 1, pa, hi, lo);
        s_hi[tid] = hi;
        s_lo[tid] = lo;
    }
    __syncthreads();
    if (tid < n) {
        const uint64_t hi = s_hi[tid], lo = s_lo[tid];
        int rk = 0;
#pragma unroll 8
        for (int q = 0; q < n; ++q) {
            const uint64_t h = s_hi[q], l = s_lo[q];
            rk += (int)(h > hi) | ((int)(h == hi) & (int)(l > lo));
        }
        if (rk < NE) {
            t.frontier[(int64_t)b * NE + rk] = cb + tid;
            t.fr_parent[(int64_t)b * NE + rk] = tid / K;
            t.fr_token[(int64_t)b * NE + rk] = tok;
        }
    }
}

}  // namespace rheo
