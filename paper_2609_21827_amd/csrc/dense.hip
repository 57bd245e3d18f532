// Level expansion over the full vocabulary (dense mode: the support is all
// of V; Sec. 3.2 before its sparse approximation).
//
// Three kernels per level:
//  * k_select (expand.hip) with list length kk = min(V, m + K): the exact
//    top-kk of every chunk by (logit desc, id asc).
//  * k_dweights, one 256-thread block per (chunk, row): merges the row's
//    chunk lists (its top-kk by logit: the maximum M and a guess of x_{m+1}),
//    then computes for every token the construction weight w1 (relative to
//    M) and the tail weight q (relative to the guessed x_{m+1}, temperature
//    T): the chunk's sums of both, the totals of q per 64-vector sub-chunk
//    (the inverse CDF's coarse level), and a flag if a token outside the
//    top-kk ties the kk-th construction weight with a smaller id (then the
//    rank by (w1 desc, id asc) is not the rank by logit).
//  * k_dpool, one 256-thread block per row: ranks the top-kk by (w1 desc, id
//    asc) -- exactly, by a row scan, when flagged -- checks the guess of
//    x_{m+1} (recomputing the tail totals when it was wrong), removes the
//    leads from the tail, samples Y by inverse CDF over token ids (sub-chunk
//    totals, then one re-read sub-chunk), forms the pool (App. C.1) and
//    stores what verification needs (Z_q, the logit of x_{m+1}, the leads).
//    Then the frontier selection shared with the sparse pool.
#include "rheo_device.h"
#include "rheo_state.h"
#include "pool_common.h"

namespace rheo {

constexpr int NTD = 256;
constexpr int KKMAX = 32;         // m + K <= 29
constexpr int DLIST_MAX = 512;    // C * kk keys a row's chunk lists hold
constexpr int NCHMAX = 1024;      // sub-chunks per row: V <= 262143, >= 256 tokens each

template <int DT>
__device__ __forceinline__ float delem(const uint4& v, int k) {
    const uint32_t* w = &v.x;
    if (DT) return (k & 1) ? bf_hi(w[k >> 1]) : bf_lo(w[k >> 1]);
    return __uint_as_float(w[k]);
}

template <int DT>
__device__ __forceinline__ uint4 dload_vec(const char* base, int vi, int V) {
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

template <int DT>
__device__ __forceinline__ float dlogit(const char* row, int v) {
    if (DT) return __uint_as_float((uint32_t)((const uint16_t*)row)[v] << 16);
    return ((const float*)row)[v];
}

// The row's top-kk by logit key from its C chunk lists (unique keys; 0 marks
// an empty slot), into s_tl[0..kk).  All threads of the block take part.
__device__ __forceinline__ void row_top_by_logit(const TreeDev& t, int row, uint64_t* s_list,
                                                 uint64_t* s_tl) {
    const int kk = t.Sc, nl = t.C * kk;
    const uint64_t* src = t.sel + (int64_t)row * nl;
    for (int i = threadIdx.x; i < nl; i += blockDim.x) s_list[i] = src[i];
    __syncthreads();
    for (int i = threadIdx.x; i < nl; i += blockDim.x) {
        const uint64_t k = s_list[i];
        if (k == 0ull) continue;
        int rk = 0;
        for (int q = 0; q < nl; ++q) rk += (int)(s_list[q] > k);
        if (rk < kk) s_tl[rk] = k;
    }
    __syncthreads();
}

// ---------------------------------------------------------------------------
// k_dweights: weights, sums and sub-chunk totals of one chunk of one row
// ---------------------------------------------------------------------------
template <int DT, int NVC>
__global__ __launch_bounds__(NTD) void k_dweights(TreeDev t, LevelArgs a) {
    constexpr int VEC = DT ? 8 : 4;
    constexpr int ESZ = DT ? 2 : 4;
    __shared__ uint64_t s_list[DLIST_MAX];
    __shared__ uint64_t s_tl[KKMAX];
    __shared__ uint32_t s_tw[KKMAX];
    __shared__ uint64_t s_red[NTD / WAVE];
    __shared__ float s_M, s_ref;
    __shared__ uint32_t s_wmin;
    __shared__ uint64_t s_kb;
    __shared__ int s_idmax;

    const int tid = threadIdx.x, lane = tid % WAVE, wid = tid / WAVE;
    const int c = blockIdx.x, row = blockIdx.y;
    const int V = t.V, m = t.m, kk = t.Sc;
    const int v0 = c * NTD * NVC;
    const char* base = (const char*)a.logits + (int64_t)row * t.stride * ESZ;

    uint4 r[NVC];
#pragma unroll
    for (int i = 0; i < NVC; ++i) r[i] = dload_vec<DT>(base, v0 + i * NTD + tid, V);

    row_top_by_logit(t, row, s_list, s_tl);
    if (tid < kk) s_tw[tid] = cweight(key_value(s_tl[tid]), key_value(s_tl[0]), a.k1);
    __syncthreads();
    if (tid == 0) {
        s_M = key_value(s_tl[0]);
        s_ref = key_value(s_tl[m]);                    // guess of x_{m+1}
        const uint32_t wmin = s_tw[kk - 1];
        int idmax = -1;
        for (int i = 0; i < kk; ++i)
            if (s_tw[i] == wmin) idmax = max(idmax, key_id(s_tl[i]));
        s_wmin = wmin;
        s_kb = s_tl[kk - 1];
        s_idmax = idmax;
    }
    __syncthreads();
    const float M = s_M, ref = s_ref;
    const uint32_t wmin = s_wmin;
    const uint64_t kb = s_kb;
    const int idmax = s_idmax;

    // Per element: w1 relative to the row maximum (never above it, so no
    // upper clamp), q relative to the guess of x_{m+1}; weights are summed
    // in pairs in 32 bits (each <= 2^30) before the 64-bit totals.  Each
    // vector's q total goes to LDS, and the totals of the sub-chunks (64
    // consecutive vectors: one wave's at one step) are formed there.  A
    // weight equal to the kk-th one is only marked per element; the exact
    // test of the rank tie runs for the marked elements alone (rare).
    uint64_t s1 = 0, zq = 0;
    bool flag = false;
    constexpr int NG = NVC < 16 ? NVC : 16;          // vectors per LDS round
    __shared__ uint64_t s_vq[NG][NTD];
    for (int g0 = 0; g0 < NVC; g0 += NG) {
#pragma unroll
        for (int ii = 0; ii < NG; ++ii) {
            const int i = g0 + ii;
            const int e0 = (v0 + i * NTD + tid) * VEC;
            // (elements past V read as -inf: weight 0 on both counts, and
            // no tie, since idmax < V)
            uint64_t sq = 0;
            uint32_t hit = 0;
#pragma unroll
            for (int k = 0; k < VEC; k += 2) {
                const float la = delem<DT>(r[i], k), lb = delem<DT>(r[i], k + 1);
                const uint32_t wa = cweight_below(la, M, a.k1);
                const uint32_t wb = cweight_below(lb, M, a.k1);
                s1 += (uint64_t)(wa + wb);
                sq += (uint64_t)(cweight(la, ref, a.kT) + cweight(lb, ref, a.kT));
                hit |= (uint32_t)(wa == wmin) << k;
                hit |= (uint32_t)(wb == wmin) << (k + 1);
            }
            if (hit) {
#pragma unroll
                for (int k = 0; k < VEC; ++k) {
                    const int id = e0 + k;
                    if (((hit >> k) & 1u) && id < idmax &&
                        logit_key(delem<DT>(r[i], k), (uint32_t)id) < kb)
                        flag = true;
                }
            }
            zq += sq;
            s_vq[ii][tid] = sq;
        }
        __syncthreads();
        // sub-chunk (ii, wave w): lanes 64 w .. 64 w + 63 of row ii, summed
        // by 4 threads of 16 entries each
        for (int q = tid; q < NG * (NTD / WAVE) * 4; q += NTD) {
            const int part = q & 3, sc = q >> 2;
            const int ii = sc / (NTD / WAVE), w = sc % (NTD / WAVE);
            uint64_t x = 0;
#pragma unroll
            for (int l = 0; l < 16; ++l) x += s_vq[ii][w * WAVE + part * 16 + l];
            x += __shfl_xor(x, 1);
            x += __shfl_xor(x, 2);
            const int sub = (v0 + (g0 + ii) * NTD) / WAVE + w;
            if (part == 0 && sub < t.NCH) t.dq[(int64_t)row * t.NCH + sub] = x;
        }
        __syncthreads();
    }
    s1 = block_sum_u64<NTD>(s1, s_red);
    zq = block_sum_u64<NTD>(zq, s_red);
    if (__syncthreads_or(flag) && tid == 0) atomicOr(&t.dflag[row], 1);
    if (tid == 0) {
        t.dpart[((int64_t)row * t.C + c) * 2 + 0] = s1;
        t.dpart[((int64_t)row * t.C + c) * 2 + 1] = zq;
    }
}

// ---------------------------------------------------------------------------
// k_dpool: ranks, tail, Y, pool and frontier of one row
// ---------------------------------------------------------------------------
template <int DT>
__global__ __launch_bounds__(NTD) void k_dpool(TreeDev t, LevelArgs a) {
    constexpr int VEC = DT ? 8 : 4;
    constexpr int ESZ = DT ? 2 : 4;
    constexpr int CHT = WAVE * VEC;              // tokens per sub-chunk
    __shared__ uint64_t s_list[DLIST_MAX];
    __shared__ uint64_t s_tl[KKMAX];             // top-kk by logit key
    __shared__ uint64_t s_x[KKMAX];              // x_1..x_kk (logit keys) by (w1 desc, id asc)
    __shared__ uint32_t s_xw[KKMAX];             // their construction weights
    __shared__ uint64_t s_rk[KKMAX];             // ranking keys (w1 << 32 | ~id)
    __shared__ uint64_t s_sub[NCHMAX];           // tail totals per sub-chunk
    __shared__ uint64_t s_cq[CHT];               // tail weights of one sub-chunk
    __shared__ uint64_t s_red[NTD / WAVE];
    __shared__ int s_pu, s_cs, s_y, s_flag, s_cnt;
    __shared__ uint64_t s_u, s_t2, s_qy;

    const int tid = threadIdx.x, lane = tid % WAVE;
    const int row = blockIdx.x;
    const int b = row / a.P, j = row % a.P;
    const int V = t.V, K = t.K, m = t.m, kk = t.Sc, C = t.C, NE = t.NE, NCH = t.NCH;
    const int level = a.level;
    const int64_t nb = (int64_t)b * t.NN;
    const char* base = (const char*)a.logits + (int64_t)row * t.stride * ESZ;

    if (tid == 0) {
        int pu = (level == 0) ? 0 : t.frontier[(int64_t)b * NE + j];
        const int lo_uid = (level == 0) ? 0 : ((level == 1) ? 1 : 1 + K + (level - 2) * NE * K);
        const int hi_uid = (level == 0) ? 1 : lo_uid + ((level == 1) ? 1 : NE) * K;
        bool bad = pu < lo_uid || pu >= hi_uid;
        if (bad) {
            atomicOr(t.err, 16);
            pu = 0;
        }
        s_pu = pu;
        // the draw of the parent's sampled slot, keyed by the launch that
        // created the parent
        s_u = philox_draw((level == 0 || bad) ? a.rng_key : a.fr_key, P_DRAFT, (uint64_t)b,
                          (uint64_t)pu);
        s_flag = t.dflag[row];
        t.dflag[row] = 0;                        // clean for the next level
        s_y = -1;
        s_cs = -1;
    }
    // the row's construction and tail totals and its sub-chunk tail totals
    // (relative to the guess of x_{m+1}), loaded now: they arrive while the
    // top of the row is ranked
    uint64_t S1 = 0, Zq = 0;
    for (int c = 0; c < C; ++c) {
        S1 += t.dpart[((int64_t)row * C + c) * 2 + 0];
        Zq += t.dpart[((int64_t)row * C + c) * 2 + 1];
    }
    uint64_t dqv[NCHMAX / NTD];
#pragma unroll
    for (int q = 0; q < NCHMAX / NTD; ++q) {
        const int i = tid + q * NTD;
        dqv[q] = (i < NCH) ? t.dq[(int64_t)row * NCH + i] : 0ull;
    }
    row_top_by_logit(t, row, s_list, s_tl);
    const float M = key_value(s_tl[0]);

    // x_1..x_kk by (w1 desc, id asc)
    if (!s_flag) {
        if (tid < kk) {
            const uint32_t w = cweight(key_value(s_tl[tid]), M, a.k1);
            s_rk[tid] = ((uint64_t)w << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)key_id(s_tl[tid]));
        }
        __syncthreads();
        if (tid < kk) {
            const uint64_t k = s_rk[tid];
            int rk = 0;
            for (int q = 0; q < kk; ++q) rk += (int)(s_rk[q] > k);
            s_x[rk] = s_tl[tid];
            s_xw[rk] = (uint32_t)(k >> 32);
        }
    } else {
        // A token outside the top-kk by logit ties the kk-th construction
        // weight with a smaller id.  The top-kk by (w1, id) is then: every
        // token with w1 above that weight (all among the top-kk by logit),
        // and the lowest ids with exactly that weight, found by a scan of
        // the row in id order (each thread a contiguous range).
        if (tid < kk) {
            const uint32_t w = cweight(key_value(s_tl[tid]), M, a.k1);
            s_rk[tid] = ((uint64_t)w << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)key_id(s_tl[tid]));
        }
        __syncthreads();
        uint32_t wmin = 0xFFFFFFFFu;
        for (int q = 0; q < kk; ++q) wmin = min(wmin, (uint32_t)(s_rk[q] >> 32));
        int ngt = 0;
        for (int q = 0; q < kk; ++q) ngt += (int)((uint32_t)(s_rk[q] >> 32) > wmin);
        const int need = kk - ngt;
        const int per = (V + NTD - 1) / NTD;
        const int lo = min(V, tid * per), hi = min(V, lo + per);
        int mine = 0;
        for (int v = lo; v < hi; ++v) mine += (int)(cweight(dlogit<DT>(base, v), M, a.k1) == wmin);
        uint64_t tot;
        int before = (int)block_excl_scan_u64<NTD>((uint64_t)mine, s_red, &tot);
        if (tid == 0) s_cnt = 0;
        __syncthreads();
        // the tokens above wmin keep their (w1, id) order first
        if (tid < kk && (uint32_t)(s_rk[tid] >> 32) > wmin) {
            const uint64_t k = s_rk[tid];
            int rk = 0;
            for (int q = 0; q < kk; ++q) rk += (int)(s_rk[q] > k);
            s_x[rk] = s_tl[tid];
            s_xw[rk] = (uint32_t)(k >> 32);
        }
        for (int v = lo; v < hi && before < need; ++v) {
            const float l = dlogit<DT>(base, v);
            if (cweight(l, M, a.k1) == wmin) {
                s_x[ngt + before] = logit_key(l, (uint32_t)v);
                s_xw[ngt + before] = wmin;
                ++before;
            }
        }
    }
    __syncthreads();

    // x_{m+1} and the tail totals
    const float ref_t = key_value(s_x[m]);
    if (tid == 0 && !(ref_t > -INFINITY)) atomicOr(t.err, 512);   // x_{m+1} is -inf
    const int nch = NCH;
    if (ref_t == key_value(s_tl[m])) {
#pragma unroll
        for (int q = 0; q < NCHMAX / NTD; ++q)
            if (tid + q * NTD < nch) s_sub[tid + q * NTD] = dqv[q];
    } else {
        // the guess of x_{m+1} was wrong (construction-weight ties): tail
        // totals again, relative to the right logit, one sub-chunk per wave
        // pass
        uint64_t part = 0;
        for (int i = tid / WAVE; i < nch; i += NTD / WAVE) {
            const int v0 = i * CHT + lane * VEC;
            uint64_t sq = 0;
            for (int k = 0; k < VEC; ++k)
                if (v0 + k < V) sq += cweight(dlogit<DT>(base, v0 + k), ref_t, a.kT);
            const uint64_t ws = wave_sum_u64(sq);
            if (lane == 0) s_sub[i] = ws;
            part += (lane == 0) ? ws : 0ull;
        }
        Zq = block_sum_u64<NTD>(part, s_red);
    }
    __syncthreads();
    // the leads leave the tail
    uint64_t lead_q = 0;
    for (int i = 0; i < m; ++i) lead_q += cweight(key_value(s_x[i]), ref_t, a.kT);
    if (tid == 0) {
        for (int i = 0; i < m; ++i) {
            const int id = key_id(s_x[i]);
            s_sub[id / CHT] -= cweight(key_value(s_x[i]), ref_t, a.kT);
        }
    }
    Zq -= lead_q;
    __syncthreads();

    // Y ~ q~_T: t = floor(U64 Zq / 2^64), the sub-chunk holding t, then the
    // first token of it whose inclusive prefix exceeds the remainder
    {
        const uint64_t tt = __umul64hi(s_u, Zq);
        const int cpt = (nch + NTD - 1) / NTD;
        const int ca = min(nch, tid * cpt), cz = min(nch, ca + cpt);
        uint64_t mysum = 0;
        for (int i = ca; i < cz; ++i) mysum += s_sub[i];
        uint64_t tot;
        uint64_t acc = block_excl_scan_u64<NTD>(mysum, s_red, &tot);
        if (acc <= tt && tt < acc + mysum) {
            for (int i = ca; i < cz; ++i) {
                if (tt < acc + s_sub[i]) {
                    s_cs = i;
                    s_t2 = tt - acc;
                    break;
                }
                acc += s_sub[i];
            }
        }
        __syncthreads();
        const int cs = s_cs;
        if (cs < 0) {
            if (tid == 0) atomicOr(t.err, 1);
        } else {
            for (int i = tid; i < CHT; i += NTD) {
                const int v = cs * CHT + i;
                uint64_t w = 0;
                if (v < V) {
                    w = cweight(dlogit<DT>(base, v), ref_t, a.kT);
                    for (int q = 0; q < m; ++q)
                        if (key_id(s_x[q]) == v) w = 0;
                }
                s_cq[i] = w;
            }
            __syncthreads();
            constexpr int TPT = CHT / NTD;       // tokens per thread (1 or 2)
            uint64_t mine = 0;
#pragma unroll
            for (int q = 0; q < TPT; ++q) mine += s_cq[tid * TPT + q];
            uint64_t acc2 = block_excl_scan_u64<NTD>(mine, s_red, &tot);
            const uint64_t t2 = s_t2;
            if (acc2 <= t2 && t2 < acc2 + mine) {
#pragma unroll
                for (int q = 0; q < TPT; ++q) {
                    const uint64_t w = s_cq[tid * TPT + q];
                    if (t2 < acc2 + w) {
                        s_y = cs * CHT + tid * TPT + q;
                        s_qy = w;
                        break;
                    }
                    acc2 += w;
                }
            }
        }
        __syncthreads();
    }
    int ytok = s_y;
    uint64_t qy = s_qy;
    if (ytok < 0) {                              // unreachable fallback
        if (tid == 0) atomicOr(t.err, 1);
        ytok = key_id(s_x[m]);
        qy = 1;
    }

    // the K children: top-m leads, Y, fills (App. C.1)
    const int pu = s_pu;
    const int cb = (level == 0) ? 1 : 1 + K + (level - 1) * NE * K;
    const int e_idx = (level == 0) ? 0 : 1 + (level - 1) * NE + j;
    if (tid == 0) {
        t.zq[(int64_t)b * t.E + e_idx] = Zq;
        t.dref[(int64_t)b * t.E + e_idx] = ref_t;
        for (int i = 0; i < m; ++i) t.dleads[((int64_t)b * t.E + e_idx) * 16 + i] = key_id(s_x[i]);
        t.first_child[nb + pu] = cb + j * K;
        t.exp_of[nb + pu] = e_idx;
        if (level == 0) emit_root(t, nb);
    }
    if (tid < K) {
        const int s = tid;
        int yr = kk;                             // Y's place among x_{m+1}.. (kk: beyond)
        for (int q = m; q < kk; ++q)
            if (key_id(s_x[q]) == ytok) yr = q;
        int kind, tok;
        double proxy;
        const double dS1 = (double)S1;
        if (s < m || t.topk) {                   // a lead (pure top-K pools: every slot)
            kind = LEAD;
            tok = key_id(s_x[s]);
            proxy = __ddiv_rn((double)s_xw[s], dS1);
        } else if (s == m) {
            kind = SAMPLED;
            tok = ytok;
            if (m >= 1) {
                uint64_t lead = 0;
                for (int q2 = 0; q2 < m; ++q2) lead += s_xw[q2];
                const uint64_t z = S1 - lead;
                const uint64_t wm = s_xw[m - 1];
                proxy = __ddiv_rn((double)(wm < z ? wm : z), dS1);
            } else {
                proxy = fmin(1.0, __dadd_rn(__ddiv_rn((double)s_xw[0], dS1), t.eps));
            }
        } else {
            const int f = s - m - 1;
            const int rk = m + f + ((m + f) >= yr ? 1 : 0);
            kind = FILL;
            tok = key_id(s_x[rk]);
            proxy = __ddiv_rn((double)s_xw[rk], dS1);
        }
        const double qtrue = (kind == SAMPLED) ? __ddiv_rn((double)qy, (double)Zq) : proxy;
        emit_child(t, level, nb, pu, parent_rec(t, level, nb, pu), cb + j * K + s, s, kind, tok,
                   proxy, qtrue, -1);
    }
    // the next frontier: the last row of the sequence to finish selects it
    select_frontier(t, a, b, s_sub, s_sub + 256);
}

template <int DT>
static void launch_dense_dt(const TreeDev& t, const LevelArgs& a, int nvc, int rows,
                            hipStream_t s) {
    const dim3 grid(t.C, rows);
    switch (nvc) {
    case 4: k_dweights<DT, 4><<<grid, NTD, 0, s>>>(t, a); break;
    case 8: k_dweights<DT, 8><<<grid, NTD, 0, s>>>(t, a); break;
    case 16: k_dweights<DT, 16><<<grid, NTD, 0, s>>>(t, a); break;
    default: k_dweights<DT, 32><<<grid, NTD, 0, s>>>(t, a); break;
    }
    k_dpool<DT><<<rows, NTD, 0, s>>>(t, a);
}

hipError_t launch_dense(const TreeDev& t, const LevelArgs& a, int nvc, hipStream_t s) {
    const int rows = t.B * a.P;
    if (t.dtype) launch_dense_dt<1>(t, a, nvc, rows, s);
    else launch_dense_dt<0>(t, a, nvc, rows, s);
    return hipGetLastError();
}

}  // namespace rheo
