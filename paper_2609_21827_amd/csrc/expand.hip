// Level expansion of the draft tree: top-S selection over each draft-logit
// row, the node's distributions, the hybrid candidate pool with its proxy and
// true probabilities, and the next frontier.
//
// One block handles one segment of one row (rows = B * P frontier nodes).
// Phase 1 (every block): stream the segment once into registers with 16-byte
// loads, take each thread's maximum, and use the S-th largest per-thread
// maximum as a threshold: at least S elements reach it, so the segment's
// top-S are all among the (typically ~1.2 S) elements at or above it.  They
// are collected in LDS and ranked exactly by (logit desc, id asc).
// Phase 2 (last block of a row): merge the segments' top-S, then build the
// pool (Sec. 3.2; App. C.1) from the truncated distribution (Sec. 3.2,
// sparse draft): construction weights q (untempered, Sec. 5.4), rank by
// (q desc, id asc), tail q~_T = q_T / z on the support minus the top-m,
// Y ~ q~_T by inverse CDF over token ids, fills, proxies
// (min{q(x_m), z}; q(x_1) + eps for m = 0), true probability q~(Y), path
// scores (App. C.1).
// Phase 3 (last row of a sequence): the n_expand children with the highest
// priority become the next frontier (Sec. 2.1; App. C.4 "expands exactly
// the K nodes with highest path scores").
#include "rheo_device.h"
#include "rheo_state.h"

namespace rheo {

constexpr int CAP = 1024;    // LDS candidate capacity (keys)
constexpr int SMAX = 1024;   // largest support

template <int DT>
__device__ __forceinline__ float elem(const uint4& v, int k) {
    const uint32_t* w = &v.x;
    if (DT) return (k & 1) ? bf_hi(w[k >> 1]) : bf_lo(w[k >> 1]);
    return __uint_as_float(w[k]);
}

// Number of keys in keys[0..n) strictly greater than k.
__device__ __forceinline__ int count_greater(const uint64_t* keys, int n, uint64_t k) {
    int r = 0;
    for (int j = 0; j < n; ++j) r += keys[j] > k;
    return r;
}

template <int NT>
__device__ void bitonic_desc(float* s) {
    for (int k = 2; k <= NT; k <<= 1) {
        for (int j = k >> 1; j > 0; j >>= 1) {
            const int i = threadIdx.x;
            const int p = i ^ j;
            if (p > i) {
                const float x = s[i], y = s[p];
                const bool desc = (i & k) == 0;
                if (desc ? (x < y) : (x > y)) { s[i] = y; s[p] = x; }
            }
            __syncthreads();
        }
    }
}

template <int DT, int NT, int EPT>
__global__ __launch_bounds__(NT) void k_expand(TreeDev t, LevelArgs a) {
    constexpr int VEC = DT ? 8 : 4;
    constexpr int NV = EPT / VEC;
    constexpr int ESZ = DT ? 2 : 4;
    static_assert(EPT % VEC == 0, "EPT must be a multiple of the vector width");

    __shared__ uint64_t s_keys[CAP];
    __shared__ uint64_t s_top[SMAX];
    __shared__ float s_sort[NT];
    __shared__ uint32_t s_w1[SMAX];
    __shared__ uint32_t s_q[SMAX];
    __shared__ int16_t s_xs[SMAX];
    __shared__ int16_t s_rank[SMAX];
    __shared__ uint64_t s_red[NT / WAVE];
    __shared__ int s_redi[NT / WAVE];
    __shared__ int s_cnt, s_last, s_y;
    __shared__ uint64_t s_t;

    const int tid = threadIdx.x;
    const int lane = tid % WAVE;
    const int row = blockIdx.x / a.G;
    const int seg = blockIdx.x % a.G;
    const int b = row / a.P;
    const int j = row % a.P;
    const int V = t.V, S = t.S, K = t.K, m = t.m;
    const int s0 = seg * a.seg_len;
    const int s1 = min(V, s0 + a.seg_len);
    const char* base = (const char*)a.logits + ((int64_t)row * t.stride + s0) * ESZ;

    // ---- phase 1: load the segment, per-thread maxima -------------------
    uint4 r[NV];
    float tmax = -INFINITY;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
        const int e = (i * NT + tid) * VEC;
        if (s0 + e + VEC <= s1) {
            r[i] = *(const uint4*)(base + (int64_t)e * ESZ);
        } else {
            uint32_t w[4];
            if (DT) {
                const uint16_t* p16 = (const uint16_t*)base;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int e0 = e + 2 * q, e1 = e0 + 1;
                    const uint32_t lo = (s0 + e0 < s1) ? p16[e0] : 0xFF80u;
                    const uint32_t hi = (s0 + e1 < s1) ? p16[e1] : 0xFF80u;
                    w[q] = lo | (hi << 16);
                }
            } else {
                const uint32_t* p32 = (const uint32_t*)base;
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    w[q] = (s0 + e + q < s1) ? p32[e + q] : 0xFF800000u;
            }
            r[i] = make_uint4(w[0], w[1], w[2], w[3]);
        }
#pragma unroll
        for (int k = 0; k < VEC; ++k) tmax = fmaxf(tmax, elem<DT>(r[i], k));
    }

    s_sort[tid] = tmax;
    if (tid == 0) s_cnt = 0;
    __syncthreads();
    bitonic_desc<NT>(s_sort);
    const float tau = (S <= NT) ? s_sort[S - 1] : -INFINITY;

    // ---- collect the candidates >= tau (wave-aggregated append) ----------
    int mine = 0;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
#pragma unroll
        for (int k = 0; k < VEC; ++k) {
            const int id = s0 + (i * NT + tid) * VEC + k;
            mine += (id < s1) && (elem<DT>(r[i], k) >= tau);
        }
    }
    {
        const int ex = wave_excl_scan(mine);
        const int tot = __shfl(ex + mine, WAVE - 1);
        int wb = 0;
        if (lane == 0 && tot) wb = atomicAdd(&s_cnt, tot);
        wb = __shfl(wb, 0);
        if (mine) {
            int pos = wb + ex;
#pragma unroll
            for (int i = 0; i < NV; ++i) {
#pragma unroll
                for (int k = 0; k < VEC; ++k) {
                    const int id = s0 + (i * NT + tid) * VEC + k;
                    const float v = elem<DT>(r[i], k);
                    if (id < s1 && v >= tau) {
                        if (pos < CAP) s_keys[pos] = logit_key(v, (uint32_t)id);
                        ++pos;
                    }
                }
            }
        }
    }
    __syncthreads();
    int c = s_cnt;

    if (c > CAP) {
        // Degenerate row (massive ties at the threshold): find the S-th
        // largest selection key exactly by bisection on the 64-bit key.
        uint64_t x = 0;
        for (int bit = 63; bit >= 0; --bit) {
            const uint64_t cand = x | (1ull << bit);
            int n = 0;
#pragma unroll
            for (int i = 0; i < NV; ++i) {
#pragma unroll
                for (int k = 0; k < VEC; ++k) {
                    const int id = s0 + (i * NT + tid) * VEC + k;
                    n += (id < s1) && (logit_key(elem<DT>(r[i], k), (uint32_t)id) >= cand);
                }
            }
            n = block_sum_i32<NT>(n, s_redi);
            if (n >= S) x = cand;
        }
        __syncthreads();
        if (tid == 0) s_cnt = 0;
        __syncthreads();
#pragma unroll
        for (int i = 0; i < NV; ++i) {
#pragma unroll
            for (int k = 0; k < VEC; ++k) {
                const int id = s0 + (i * NT + tid) * VEC + k;
                if (id < s1) {
                    const uint64_t key = logit_key(elem<DT>(r[i], k), (uint32_t)id);
                    if (key >= x) {
                        const int pos = atomicAdd(&s_cnt, 1);
                        if (pos < CAP) s_keys[pos] = key;
                    }
                }
            }
        }
        __syncthreads();
        c = min(s_cnt, CAP);
    }

    // ---- exact top-S of the candidates, sorted -------------------------
    int ns = min(S, c);
    for (int i = tid; i < c; i += NT) {
        const uint64_t key = s_keys[i];
        const int rk = count_greater(s_keys, c, key);
        if (rk < ns) s_top[rk] = key;
    }
    __syncthreads();

    // ---- merge the segments of the row ----------------------------------
    if (a.G * S > CAP) {                 // excluded by the host's launch shape
        if (tid == 0) atomicOr(t.err, 64);
        return;
    }
    if (a.G > 1) {
        uint64_t* out = t.seg_keys + ((int64_t)row * a.G + seg) * S;
        for (int i = tid; i < S; i += NT) out[i] = (i < ns) ? s_top[i] : 0ull;
        __threadfence();
        __syncthreads();
        if (tid == 0) s_last = (atomicAdd(&t.row_cnt[row], 1u) == (uint32_t)(a.G - 1));
        __syncthreads();
        if (!s_last) return;
        __threadfence();
        if (tid == 0) t.row_cnt[row] = 0u;
        const uint64_t* in = t.seg_keys + (int64_t)row * a.G * S;
        const int n = a.G * S;
        for (int i = tid; i < n; i += NT) s_keys[i] = in[i];
        __syncthreads();
        for (int i = tid; i < n; i += NT) {
            const uint64_t key = s_keys[i];
            if (key == 0ull) continue;
            const int rk = count_greater(s_keys, n, key);
            if (rk < S) s_top[rk] = key;
        }
        ns = S;
        __syncthreads();
    }

    // ---- phase 2: the node's distributions and its pool -----------------
    const int level = a.level;
    const int NE = t.NE, NN = t.NN;
    const int64_t nb = (int64_t)b * NN;
    int pu = (level == 0) ? 0 : t.frontier[b * NE + j];
    if (pu < 0 || pu >= NN) {
        if (tid == 0) atomicOr(t.err, 16);
        pu = 0;
    }
    const int cb = (level == 0) ? 1 : 1 + K + (level - 1) * NE * K;
    const int e_idx = (level == 0) ? 0 : 1 + (level - 1) * NE + j;
    double pscore = 1.0;
    uint64_t ppath = 0;
    if (level > 0) {
        pscore = t.score[nb + pu];
        ppath = t.path[nb + pu];
    }

    const float M = key_value(s_top[0]);
    uint64_t part = 0;
    for (int i = tid; i < ns; i += NT) {
        const uint32_t w = cweight(key_value(s_top[i]), M, a.k1);
        s_w1[i] = w;
        part += w;
    }
    const uint64_t S1 = block_sum_u64<NT>(part, s_red);
    // rank by construction weight (desc), then id (asc)
    for (int i = tid; i < ns; i += NT)
        s_keys[i] = ((uint64_t)s_w1[i] << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)key_id(s_top[i]));
    __syncthreads();
    for (int i = tid; i < ns; i += NT) {
        const int rk = count_greater(s_keys, ns, s_keys[i]);
        s_xs[rk] = (int16_t)i;
        s_rank[i] = (int16_t)rk;
    }
    __syncthreads();
    const float ref_t = key_value(s_top[s_xs[m]]);
    part = 0;
    for (int i = tid; i < ns; i += NT) {
        uint32_t q = 0;
        if (s_rank[i] >= m) q = cweight(key_value(s_top[i]), ref_t, a.kT);
        s_q[i] = q;
        part += q;
    }
    const uint64_t Zq = block_sum_u64<NT>(part, s_red);
    if (tid == 0) {
        const uint64_t u = philox_draw(a.rng_key, P_DRAFT, (uint64_t)b, (uint64_t)pu);
        s_t = __umul64hi(u, Zq);
        s_y = -1;
    }
    __syncthreads();
    const uint64_t tt = s_t;
    const int64_t tail_base = ((int64_t)b * t.E + e_idx) * S;
    for (int i = tid; i < ns; i += NT) {
        if (s_rank[i] < m) continue;
        const int id = key_id(s_top[i]);
        uint64_t pre = 0;
        int idr = 0;
        for (int q = 0; q < ns; ++q) {
            if (s_rank[q] < m) continue;
            if (key_id(s_top[q]) < id) { pre += s_q[q]; ++idr; }
        }
        if (pre <= tt && tt < pre + s_q[i]) s_y = i;
        t.tail_id[tail_base + idr] = id;
        t.tail_q[tail_base + idr] = s_q[i];
    }
    __syncthreads();
    int yi = s_y;
    if (yi < 0) {                      // unreachable: t < Zq always has an owner
        if (tid == 0) atomicOr(t.err, 1);
        yi = s_xs[m];
    }
    const int yrank = s_rank[yi];
    if (tid == 0) {
        t.zq[(int64_t)b * t.E + e_idx] = Zq;
        t.first_child[nb + pu] = cb + j * K;
        t.exp_of[nb + pu] = e_idx;
        if (level == 0) {
            t.tok[nb] = -1;
            t.par[nb] = -1;
            t.meta[nb] = 0;
            t.proxy[nb] = 1.0;
            t.qtrue[nb] = 1.0;
            t.score[nb] = 1.0;
            t.path[nb] = 0;
        }
    }
    if (tid < K) {
        const int s = tid;
        int item, kind;
        if (s < m) {
            item = s_xs[s];
            kind = LEAD;
        } else if (s == m) {
            item = yi;
            kind = SAMPLED;
        } else {
            const int f = s - m - 1;
            const int rk = m + f + ((m + f) >= yrank ? 1 : 0);
            item = s_xs[rk];
            kind = FILL;
        }
        double proxy;
        const double dS1 = (double)S1;
        if (kind == SAMPLED) {
            if (m >= 1) {
                uint64_t lead = 0;
                for (int q = 0; q < m; ++q) lead += s_w1[s_xs[q]];
                const uint64_t z = S1 - lead;
                const uint64_t wm = s_w1[s_xs[m - 1]];
                proxy = __ddiv_rn((double)(wm < z ? wm : z), dS1);
            } else {
                proxy = fmin(1.0, __dadd_rn(__ddiv_rn((double)s_w1[s_xs[0]], dS1), t.eps));
            }
        } else {
            proxy = __ddiv_rn((double)s_w1[item], dS1);
        }
        const double qtrue = (kind == SAMPLED) ? __ddiv_rn((double)s_q[item], (double)Zq) : proxy;
        const int uid = cb + j * K + s;
        const int64_t o = nb + uid;
        t.tok[o] = key_id(s_top[item]);
        t.par[o] = pu;
        t.meta[o] = (level + 1) | ((s + 1) << 8) | (kind << 16);
        t.proxy[o] = proxy;
        t.qtrue[o] = qtrue;
        t.score[o] = __dmul_rn(pscore, proxy);
        t.path[o] = ppath | ((uint64_t)(s + 1) << (56 - 4 * level));
        t.first_child[o] = -1;
        t.exp_of[o] = -1;
    }

    // ---- phase 3: next frontier (last row of the sequence) ---------------
    __threadfence();
    __syncthreads();
    if (tid == 0) s_last = (atomicAdd(&t.seq_cnt[b], 1u) == (uint32_t)(a.P - 1));
    __syncthreads();
    if (!s_last) return;
    __threadfence();
    if (tid == 0) t.seq_cnt[b] = 0u;
    if (level == t.D - 1) return;
    const int n = a.P * K;
    uint64_t* s_hi = s_keys;
    uint64_t* s_lo = s_top;
    for (int i = tid; i < n; i += NT) {
        const int64_t o = nb + cb + i;
        uint64_t hi, lo;
        prio_key(t.score[o], level + 1, t.path[o], hi, lo);
        s_hi[i] = hi;
        s_lo[i] = lo;
    }
    __syncthreads();
    for (int i = tid; i < n; i += NT) {
        const uint64_t hi = s_hi[i], lo = s_lo[i];
        int rk = 0;
        for (int q = 0; q < n; ++q)
            rk += (s_hi[q] > hi) || (s_hi[q] == hi && s_lo[q] > lo);
        if (rk < NE) {
            t.frontier[b * NE + rk] = cb + i;
            t.fr_parent[b * NE + rk] = i / K;
            t.fr_token[b * NE + rk] = t.tok[nb + cb + i];
        }
    }
}

// (dtype, threads, elements per thread) variants; the host picks the one
// whose segment capacity suits the vocabulary and row count.
static const ExpandVariant kVariants[2][3] = {
    {{512, 32}, {512, 64}, {256, 16}},     // fp32
    {{512, 64}, {512, 128}, {256, 32}},    // bf16
};

int expand_variant_count(int) { return 3; }
ExpandVariant expand_variant(int dtype, int v) { return kVariants[dtype ? 1 : 0][v]; }

hipError_t launch_expand(const TreeDev& t, const LevelArgs& a, int variant,
                         hipStream_t s) {
    const int rows = t.B * a.P;
    const dim3 grid(rows * a.G);
    if (t.dtype) {
        switch (variant) {
        case 0: k_expand<1, 512, 64><<<grid, 512, 0, s>>>(t, a); break;
        case 1: k_expand<1, 512, 128><<<grid, 512, 0, s>>>(t, a); break;
        default: k_expand<1, 256, 32><<<grid, 256, 0, s>>>(t, a); break;
        }
    } else {
        switch (variant) {
        case 0: k_expand<0, 512, 32><<<grid, 512, 0, s>>>(t, a); break;
        case 1: k_expand<0, 512, 64><<<grid, 512, 0, s>>>(t, a); break;
        default: k_expand<0, 256, 16><<<grid, 256, 0, s>>>(t, a); break;
        }
    }
    return hipGetLastError();
}

}  // namespace rheo
