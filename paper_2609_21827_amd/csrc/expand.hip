// Level expansion of the draft tree: parent selection, top-S selection over
// each draft-logit row, the node's distributions, the hybrid candidate pool
// with its proxy and true probabilities.
//
// One 1024-thread block handles one frontier row (rows = B * P), so no
// block ever waits for another:
//  * prologue (level >= 1): the block's parent is the j-th best child of the
//    previous level by priority (Sec. 2.1; App. C.4 "expands exactly the K
//    nodes with highest path scores"); it is ranked from the children records
//    the previous launch wrote, while the row loads are in flight.
//  * the row is streamed once from HBM into registers with 16-byte loads;
//    each thread keeps its maximum.  Every wave sorts its 64 maxima; with
//    c = ceil(S / waves), the smallest of the waves' c-th largest maxima is a
//    threshold that at least S elements reach, so the row's top-S (logit
//    desc, id asc) are among the elements at or above it (typically ~1.3 S).
//    They are collected in LDS and ranked exactly.
//  * the pool (Sec. 3.2; App. C.1) from the truncated distribution (Sec.
//    3.2, sparse draft): construction weights q (untempered, Sec. 5.4),
//    ranks by (q desc, id asc), tail q~_T = q_T / z on the support minus the
//    top-m, Y ~ q~_T by inverse CDF over token ids, fills, proxies
//    (min{q(x_m), z}; q(x_1) + eps for m = 0), true probability q~(Y), path
//    scores (App. C.1).  The tail is stored id-sorted for verification.
#include "rheo_device.h"
#include "rheo_state.h"

namespace rheo {

constexpr int NT = 1024;
constexpr int CAP = 1024;    // LDS candidate capacity
constexpr int SMAX = 1024;   // largest support
constexpr int NWAVE = NT / WAVE;

template <int DT>
__device__ __forceinline__ float elem(const uint4& v, int k) {
    const uint32_t* w = &v.x;
    if (DT) return (k & 1) ? bf_hi(w[k >> 1]) : bf_lo(w[k >> 1]);
    return __uint_as_float(w[k]);
}

// Element k of a vector for a k known only at run time (selects, so the
// vector stays in registers).
template <int DT>
__device__ __forceinline__ float elem_dyn(const uint4& v, int k) {
    const int wi = DT ? (k >> 1) : k;
    const uint32_t w = wi == 0 ? v.x : wi == 1 ? v.y : wi == 2 ? v.z : v.w;
    if (DT) return (k & 1) ? bf_hi(w) : bf_lo(w);
    return __uint_as_float(w);
}

// Vector vi (VEC consecutive elements) of a row; elements past V read as -inf.
template <int DT>
__device__ __forceinline__ uint4 load_row_vec(const char* base, int vi, int V) {
    constexpr int VEC = DT ? 8 : 4;
    constexpr int ESZ = DT ? 2 : 4;
    const int e = vi * VEC;
    if (e + VEC <= V) return load_stream16(base + (int64_t)e * ESZ);
    uint32_t w[4];
    if (DT) {
        const uint16_t* p16 = (const uint16_t*)base;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int e0 = e + 2 * q;
            const uint32_t lo = (e0 < V) ? p16[e0] : 0xFF80u;
            const uint32_t hi = (e0 + 1 < V) ? p16[e0 + 1] : 0xFF80u;
            w[q] = lo | (hi << 16);
        }
    } else {
        const uint32_t* p32 = (const uint32_t*)base;
#pragma unroll
        for (int q = 0; q < 4; ++q) w[q] = (e + q < V) ? p32[e + q] : 0xFF800000u;
    }
    return make_uint4(w[0], w[1], w[2], w[3]);
}

// Orders LDS accesses of the lanes of one wave (no block barrier).
__device__ __forceinline__ void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
}

template <int DT, int NV>
__global__ __launch_bounds__(NT) void k_expand(TreeDev t, LevelArgs a) {
    constexpr int VEC = DT ? 8 : 4;
    constexpr int ESZ = DT ? 2 : 4;
    constexpr int NM = DT ? (NV + 1) / 2 : NV;   // registers of per-vector maxima

    __shared__ uint64_t s_keys[CAP];
    __shared__ uint64_t s_top[SMAX];
    __shared__ uint32_t s_w1[SMAX];
    __shared__ uint32_t s_q[SMAX];
    __shared__ int16_t s_rank[SMAX];
    __shared__ int16_t s_wr[SMAX];     // support item -> rank by construction weight
    __shared__ int16_t s_xs[SMAX];     // rank by construction weight -> support item
    __shared__ int s_redi[NWAVE];
    __shared__ int s_cnt, s_y, s_pu, s_yi;
    __shared__ uint64_t s_u;

    const int tid = threadIdx.x;
    const int lane = tid % WAVE, wid = tid / WAVE;
    const int row = blockIdx.x;
    const int b = row / a.P;
    const int j = row % a.P;
    const int V = t.V, S = t.S, K = t.K, m = t.m;
    const int level = a.level;
    const int NE = t.NE, NN = t.NN;
    const int64_t nb = (int64_t)b * NN;
    const char* base = (const char*)a.logits + (int64_t)row * t.stride * ESZ;

    // ---- stream the row into registers -------------------------------------
    uint4 r[NV];
#pragma unroll
    for (int i = 0; i < NV; ++i) r[i] = load_row_vec<DT>(base, i * NT + tid, V);

    // ---- prologue: this row's parent (ranked while the loads are in flight),
    //      and the Philox draw of its sampled slot
    if (tid == 0) {
        s_cnt = 0;
        s_pu = -1;
    }
    __syncthreads();
    if (level == 0) {
        if (tid == 0) s_pu = 0;
    } else {
        const int pcb = (level == 1) ? 1 : 1 + K + (level - 2) * NE * K;
        const int n = ((level == 1) ? 1 : NE) * K;
        uint64_t* s_hi = s_keys;
        uint64_t* s_lo = s_top;
        if (tid < n) {
            const int64_t o = nb + pcb + tid;
            uint64_t hi, lo;
            prio_key(t.score[o], level, t.path[o], hi, lo);
            s_hi[tid] = hi;
            s_lo[tid] = lo;
        }
        __syncthreads();
        if (tid < n) {
            const uint64_t hi = s_hi[tid], lo = s_lo[tid];
            int rk = 0;
            for (int q = 0; q < n; ++q)
                rk += (s_hi[q] > hi) || (s_hi[q] == hi && s_lo[q] > lo);
            if (rk == j) s_pu = pcb + tid;
        }
    }
    __syncthreads();
    if (tid == 0) {
        int pu = s_pu;
        if (pu < 0 || pu >= NN) {
            atomicOr(t.err, 16);
            pu = 0;
            s_pu = 0;
        }
        s_u = philox_draw(a.rng_key, P_DRAFT, (uint64_t)b, (uint64_t)pu);
    }

    // ---- per-vector maxima (exact) and this thread's maximum ----------------
    // bf16: a packed word read as fp32 is its high element plus a fraction of
    // one bf16 ulp (the low element's bits), so the maximum over the raw words
    // and the unpacked low elements, with its low 16 bits cleared, is exactly
    // the maximum element (logits are finite; padding words are NaN and ignored)
    uint32_t vm[NM];
#pragma unroll
    for (int q = 0; q < NM; ++q) vm[q] = 0;
    float tmax = -INFINITY;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
        float mx;
        if (DT) {
            const uint32_t* w = &r[i].x;
            mx = fmaxf(fmaxf(__uint_as_float(w[0]), bf_lo(w[0])), __uint_as_float(w[1]));
            mx = fmaxf(fmaxf(mx, bf_lo(w[1])), __uint_as_float(w[2]));
            mx = fmaxf(fmaxf(mx, bf_lo(w[2])), __uint_as_float(w[3]));
            mx = fmaxf(mx, bf_lo(w[3]));
            const uint32_t hb = __float_as_uint(mx) & 0xFFFF0000u;
            mx = __uint_as_float(hb);
            vm[i / 2] |= (i & 1) ? hb : (hb >> 16);
        } else {
            mx = fmaxf(fmaxf(elem<DT>(r[i], 0), elem<DT>(r[i], 1)),
                       fmaxf(elem<DT>(r[i], 2), elem<DT>(r[i], 3)));
            vm[i] = __float_as_uint(mx);
        }
        tmax = fmaxf(tmax, mx);
    }

    // ---- threshold: each wave sorts its maxima and offers its top L; the
    //      S-th largest offered value is reached by at least S elements
    //      (usually it is the S-th largest maximum itself)
    const int L = min(WAVE, 2 * ((S + NWAVE - 1) / NWAVE));
    const float srt = wave_sort_desc(tmax);
    float* s_off = (float*)s_w1;                 // NWAVE * L <= 1024 offered values
    if (lane < L) s_off[wid * L + lane] = srt;
    __syncthreads();
    if (tid == 0) s_cnt = 0x7FFFFFFF;
    __syncthreads();
    {
        const int n = NWAVE * L;
        const int F = NT / n;                    // lanes per offered value (>= 1)
        const int i = tid / F, sub = tid % F;
        const float v = s_off[i];
        int gt = 0;
        for (int jj = sub; jj < n; jj += F) gt += s_off[jj] > v;
        for (int o = 1; o < F; o <<= 1) gt += __shfl_xor(gt, o);
        if (sub == 0 && gt < S) atomicMin(&s_cnt, (int)(ord32(v) ^ 0x80000000u));
    }
    __syncthreads();
    float tau = unord32((uint32_t)s_cnt ^ 0x80000000u);
    if (V <= CAP) tau = -INFINITY;
    __syncthreads();
    if (tid == 0) s_cnt = 0;
    __syncthreads();

    // ---- candidates >= tau: one compare per vector, a rare element scan ----
    opaque_regs(r);
#pragma unroll
    for (int i = 0; i < NV; ++i) {
        const float vmax = DT ? ((i & 1) ? bf_hi(vm[i / 2]) : bf_lo(vm[i / 2]))
                              : __uint_as_float(vm[i]);
        if (vmax >= tau) {
            const int e0 = (i * NT + tid) * VEC;
#pragma unroll
            for (int k = 0; k < VEC; ++k) {
                const float v = elem<DT>(r[i], k);
                const int id = e0 + k;
                if (v >= tau && id < V) {
                    const int pos = atomicAdd(&s_cnt, 1);
                    if (pos < CAP) s_keys[pos] = logit_key(v, (uint32_t)id);
                }
            }
        }
    }
    __syncthreads();
    int c = s_cnt;

    if (c > CAP) {
        // Degenerate row (massive ties at the threshold): the S-th largest
        // selection key, exactly, by bisection on the 64-bit key.  Rare, so
        // it re-reads the row from memory rather than holding more registers.
        const int nvec = (V + VEC - 1) / VEC;
        uint64_t x = 0;
        for (int bit = 63; bit >= 0; --bit) {
            const uint64_t cand = x | (1ull << bit);
            int n = 0;
#pragma unroll 1
            for (int vi = tid; vi < nvec; vi += NT) {
                const uint4 w = load_row_vec<DT>(base, vi, V);
#pragma unroll
                for (int k = 0; k < VEC; ++k) {
                    const int id = vi * VEC + k;
                    n += (id < V) && (logit_key(elem<DT>(w, k), (uint32_t)id) >= cand);
                }
            }
            n = block_sum_i32<NT>(n, s_redi);
            if (n >= S) x = cand;
        }
        __syncthreads();
        if (tid == 0) s_cnt = 0;
        __syncthreads();
#pragma unroll 1
        for (int vi = tid; vi < nvec; vi += NT) {
            const uint4 w = load_row_vec<DT>(base, vi, V);
#pragma unroll
            for (int k = 0; k < VEC; ++k) {
                const int id = vi * VEC + k;
                if (id < V) {
                    const uint64_t key = logit_key(elem<DT>(w, k), (uint32_t)id);
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

    // ---- exact top-S of the candidates (sorted by logit desc, id asc) -------
    rank_keys<NT>(s_keys, c, s_rank);
    __syncthreads();
    for (int i = tid; i < c; i += NT) {
        const int rk = s_rank[i];
        if (rk < S) s_top[rk] = s_keys[i];
    }
    __syncthreads();

    // ---- the node's distributions and its pool: one wave; the other waves
    //      leave, so the next row's block can start loading -------------------
    if (wid != 0) return;
    const int pu = s_pu;
    const int cb = (level == 0) ? 1 : 1 + K + (level - 1) * NE * K;
    const int e_idx = (level == 0) ? 0 : 1 + (level - 1) * NE + j;
    const int IPL = (S + WAVE - 1) / WAVE;       // support items per lane (<= 16)
    const float M = key_value(s_top[0]);
    // construction weights (untempered unless asked), S1, rank by (w1 desc, id asc)
    uint64_t part = 0;
    for (int q = 0; q < IPL; ++q) {
        const int i = q * WAVE + lane;
        if (i < S) {
            const uint64_t tk = s_top[i];
            const uint32_t w = cweight(key_value(tk), M, a.k1);
            s_w1[i] = w;
            s_keys[i] = ((uint64_t)w << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)key_id(tk));
            part += w;
        }
    }
    const uint64_t S1 = wave_sum_u64(part);
    wave_sync();
    for (int q = 0; q < IPL; ++q) {
        const int i = q * WAVE + lane;
        if (i < S) {
            const uint64_t k = s_keys[i];
            int rk = 0;
            for (int jj = 0; jj < S; ++jj) rk += s_keys[jj] > k;
            s_wr[i] = (int16_t)rk;
            s_xs[rk] = (int16_t)i;
        }
    }
    wave_sync();
    // tail q~_T (relative to x_{m+1}), its total, and its order by token id
    const float ref_t = key_value(s_top[s_xs[m]]);
    part = 0;
    for (int q = 0; q < IPL; ++q) {
        const int i = q * WAVE + lane;
        if (i < S) {
            const bool tail = s_wr[i] >= m;
            const uint64_t tk = s_top[i];
            const uint32_t w = tail ? cweight(key_value(tk), ref_t, a.kT) : 0u;
            s_q[i] = w;
            part += w;
            s_keys[i] = tail ? (uint64_t)(0xFFFFFFFFu - (uint32_t)key_id(tk)) + 1 : 0ull;
        }
    }
    const uint64_t Zq = wave_sum_u64(part);
    wave_sync();
    const int ntail = S - m;
    for (int q = 0; q < IPL; ++q) {
        const int i = q * WAVE + lane;
        if (i < S && s_keys[i] != 0ull) {
            const uint64_t k = s_keys[i];
            int rk = 0;
            for (int jj = 0; jj < S; ++jj) rk += s_keys[jj] > k;
            s_rank[i] = (int16_t)rk;              // position in id order
        }
    }
    wave_sync();
    // id-sorted tail written straight to the tree (q~ for verification) and
    // kept in LDS for the inverse CDF (s_keys is free again)
    const int64_t tail_base = ((int64_t)b * t.E + e_idx) * S;
    for (int q = 0; q < IPL; ++q) {
        const int i = q * WAVE + lane;
        if (i < S && s_wr[i] >= m) {
            const int idr = s_rank[i];
            const int id = key_id(s_top[i]);
            s_keys[idr] = ((uint64_t)(uint32_t)id << 32) | s_q[i];
            t.tail_id[tail_base + idr] = id;
            t.tail_q[tail_base + idr] = s_q[i];
        }
    }
    wave_sync();
    // Y ~ q~_T: t = floor(U64 Zq / 2^64), the first id-ordered tail entry whose
    // inclusive prefix exceeds t (each lane scans a contiguous block)
    const uint64_t tt = __umul64hi(s_u, Zq);
    const int lo = lane * IPL, hi = min(ntail, lo + IPL);
    uint64_t mysum = 0;
    for (int i = lo; i < hi; ++i) mysum += (uint32_t)s_keys[i];
    const uint64_t incl = wave_incl_scan_u64(mysum);
    uint64_t acc = incl - mysum;
    if (lane == 0) s_y = -1;
    wave_sync();
    if (acc <= tt && tt < incl) {
        for (int i = lo; i < hi; ++i) {
            const uint64_t w = (uint32_t)s_keys[i];
            if (tt < acc + w) {
                s_y = (int)(s_keys[i] >> 32);
                break;
            }
            acc += w;
        }
    }
    wave_sync();
    const int ytok = s_y;
    if (lane == 0) {
        s_yi = s_xs[m];                        // unreachable fallback
        if (ytok < 0) atomicOr(t.err, 1);
    }
    wave_sync();
    for (int q = 0; q < IPL; ++q) {
        const int i = q * WAVE + lane;
        if (i < S && s_wr[i] >= m && key_id(s_top[i]) == ytok) s_yi = i;
    }
    wave_sync();
    const int yi = s_yi;
    if (lane == 0) {
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
    // ---- the K children: top-m leads, Y, fills (App. C.1) ------------------
    if (lane < K) {
        const int s = lane;
        const int yr = s_wr[yi];
        int item, kind;
        if (s < m) {
            item = s_xs[s];
            kind = LEAD;
        } else if (s == m) {
            item = yi;
            kind = SAMPLED;
        } else {
            const int f = s - m - 1;
            const int rk = m + f + ((m + f) >= yr ? 1 : 0);
            item = s_xs[rk];
            kind = FILL;
        }
        double pscore = 1.0;
        uint64_t ppath = 0;
        if (level > 0) {
            pscore = t.score[nb + pu];
            ppath = t.path[nb + pu];
        }
        double proxy;
        const double dS1 = (double)S1;
        if (kind == SAMPLED) {
            if (m >= 1) {
                uint64_t lead = 0;
                for (int q2 = 0; q2 < m; ++q2) lead += s_w1[s_xs[q2]];
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
}

// The frontier of the last expanded level in rank order, for the caller
// (rheo_frontier): the n_expand best children by priority, per sequence.
__global__ __launch_bounds__(256) void k_frontier(TreeDev t, int level, int P) {
    __shared__ uint64_t s_hi[256], s_lo[256];
    const int b = blockIdx.x, tid = threadIdx.x;
    const int K = t.K, NE = t.NE;
    const int cb = (level == 0) ? 1 : 1 + K + (level - 1) * NE * K;
    const int n = P * K;
    const int64_t nb = (int64_t)b * t.NN;
    if (tid < n) {
        uint64_t hi, lo;
        prio_key(t.score[nb + cb + tid], level + 1, t.path[nb + cb + tid], hi, lo);
        s_hi[tid] = hi;
        s_lo[tid] = lo;
    }
    __syncthreads();
    if (tid < n) {
        const uint64_t hi = s_hi[tid], lo = s_lo[tid];
        int rk = 0;
        for (int q = 0; q < n; ++q) rk += (s_hi[q] > hi) || (s_hi[q] == hi && s_lo[q] > lo);
        if (rk < NE) {
            t.fr_parent[b * NE + rk] = tid / K;
            t.fr_token[b * NE + rk] = t.tok[nb + cb + tid];
        }
    }
}

// Registers per thread hold NV 16-byte vectors: a row must fit NT * NV * VEC.
static const int kNV[] = {1, 2, 4, 8, 12, 16, 20};

int expand_variant_count(int) { return (int)(sizeof(kNV) / sizeof(kNV[0])); }
ExpandVariant expand_variant(int dtype, int v) {
    return ExpandVariant{NT, kNV[v] * (dtype ? 8 : 4)};
}

template <int DT>
static void launch_dt(const TreeDev& t, const LevelArgs& a, int v, dim3 grid, hipStream_t s) {
    switch (v) {
    case 0: k_expand<DT, 1><<<grid, NT, 0, s>>>(t, a); break;
    case 1: k_expand<DT, 2><<<grid, NT, 0, s>>>(t, a); break;
    case 2: k_expand<DT, 4><<<grid, NT, 0, s>>>(t, a); break;
    case 3: k_expand<DT, 8><<<grid, NT, 0, s>>>(t, a); break;
    case 4: k_expand<DT, 12><<<grid, NT, 0, s>>>(t, a); break;
    case 5: k_expand<DT, 16><<<grid, NT, 0, s>>>(t, a); break;
    default: k_expand<DT, 20><<<grid, NT, 0, s>>>(t, a); break;
    }
}

hipError_t launch_expand(const TreeDev& t, const LevelArgs& a, int variant, hipStream_t s) {
    const dim3 grid(t.B * a.P);
    if (t.dtype) launch_dt<1>(t, a, variant, grid, s);
    else launch_dt<0>(t, a, variant, grid, s);
    return hipGetLastError();
}

hipError_t launch_frontier(const TreeDev& t, int level, int P, hipStream_t s) {
    k_frontier<<<t.B, 256, 0, s>>>(t, level, P);
    return hipGetLastError();
}

}  // namespace rheo
