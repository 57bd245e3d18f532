// Level expansion of the draft tree: top-S selection over each draft-logit
// row, the node's distributions, the hybrid candidate pool with its proxy
// and true probabilities, and the parent each row belongs to.
//
// Two kernels per level:
//  * k_select, one 256-thread block per (chunk, row): the chunk is streamed
//    from HBM into registers with 16-byte loads and its exact top-Sc by
//    (logit desc, id asc) is written, sorted, to the tree's selection
//    scratch (Sc = S: a chunk is larger than any support).  The row's top-S
//    lies in the union of its chunks' top-S.  Within a chunk, a value that
//    Sc per-vector maxima reach is a threshold at least Sc elements reach,
//    so the chunk's top-Sc are among the few elements at or above it; they
//    are collected in LDS and ranked exactly.  Many small blocks per CU keep
//    loads in flight while other blocks rank.
//  * k_pool, one 256-thread block per row: takes the row's parent from the
//    stored frontier, merges the chunk lists into the row's top-S support
//    (Sec. 3.2, sparse draft distributions), and forms the pool (Sec. 3.2;
//    App. C.1): construction weights q (untempered, Sec. 5.4), ranks by
//    (q desc, id asc), the tail q~_T = q_T / z on the support minus the
//    top-m, Y ~ q~_T by inverse CDF over token ids, fills, proxies
//    (min{q(x_m), z}; q(x_1) + eps for m = 0), the true probability q~(Y),
//    path scores (App. C.1).  The tail is stored id-sorted for verification.
//    The last row of a sequence to finish (an arrival counter) ranks the
//    level's new children by priority and stores the n_expand best, which
//    the next level's rows expand (Sec. 2.1; App. C.4, step 1).
// No block waits for another; children fields pass between blocks only
// through agent-coherent atomic stores and loads.
#include "rheo_device.h"
#include "rheo_state.h"
#include "pool_common.h"

namespace rheo {

constexpr int NTC = 256;      // threads per k_select block
constexpr int NTP = 256;      // threads per k_pool block
constexpr int CAPC = 1024;    // candidates a chunk collects in LDS
constexpr int CAPV = 512;     // candidate vectors a chunk collects in LDS
constexpr int SMAX = 1024;    // largest support
constexpr int MERGE_MAX = 2048;  // chunk-list keys one row merges (C * Sc)

template <int DT>
__device__ __forceinline__ float elem(const uint4& v, int k) {
    const uint32_t* w = &v.x;
    if (DT) return (k & 1) ? bf_hi(w[k >> 1]) : bf_lo(w[k >> 1]);
    return __uint_as_float(w[k]);
}

// Vector vi (VEC consecutive elements) of a row; elements past V read as the
// most negative finite value (bf16 0xFF7F, fp32 -inf).  A bf16 pair read as
// one fp32 word must never be a NaN (the maxima below compare raw words), and
// 0xFF80 (-inf) in the high half would make it one.
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
            const uint32_t lo = (e0 < V) ? p16[e0] : 0xFF7Fu;
            const uint32_t hi = (e0 + 1 < V) ? p16[e0 + 1] : 0xFF7Fu;
            w[q] = lo | (hi << 16);
        }
    } else {
        const uint32_t* p32 = (const uint32_t*)base;
#pragma unroll
        for (int q = 0; q < 4; ++q) w[q] = (e + q < V) ? p32[e + q] : 0xFF800000u;
    }
    return make_uint4(w[0], w[1], w[2], w[3]);
}

// ---------------------------------------------------------------------------
// the pool of one row, formed by the last of its chunk blocks: parent,
// support, distributions and children
// ---------------------------------------------------------------------------
// LDS layout of the pool phase inside the block's dynamic buffer; the
// previous level's priority keys (<= 225 of them) share the regions of the
// support and the ranking keys.
struct PoolLds {
    int m, top, k2, w1, q, tq, wr, xs, ir, tx, bytes;
};
__host__ __device__ inline int pad16(int x) { return (x + 15) & ~15; }
__host__ __device__ inline PoolLds pool_lds(int S, int C) {
    PoolLds L;
    const int S2 = S > 256 ? S : 256;
    L.m = 0;
    L.top = L.m + pad16(8 * C * S);
    L.k2 = L.top + pad16(8 * S2);
    L.w1 = L.k2 + pad16(8 * S2);
    L.q = L.w1 + pad16(4 * S);
    L.tq = L.q + pad16(4 * S);
    L.wr = L.tq + pad16(4 * S);
    L.xs = L.wr + pad16(2 * S);
    L.ir = L.xs + pad16(2 * S);
    L.tx = L.ir + pad16(2 * S);
    L.bytes = L.tx + pad16(2 * S);
    return L;
}

// The pool of one row from its merged support s_top (App. C.1), formed by
// NT threads (tid < NT).  Children fields the frontier selection reads in
// other blocks (token, score, path) are published with agent-scope atomics.
template <int NT>
__device__ __forceinline__ void pool_form(const TreeDev& t, const LevelArgs& a, int row,
                                          uint8_t* lds, int pu, uint64_t u, uint64_t* s_red,
                                          int* s_yi) {
    const PoolLds L = pool_lds(t.S, t.C);
    uint64_t* s_top = (uint64_t*)(lds + L.top);
    uint64_t* s_k2 = (uint64_t*)(lds + L.k2);
    uint32_t* s_w1 = (uint32_t*)(lds + L.w1);
    uint32_t* s_q = (uint32_t*)(lds + L.q);
    uint32_t* s_tq = (uint32_t*)(lds + L.tq);
    int16_t* s_wr = (int16_t*)(lds + L.wr);
    int16_t* s_xs = (int16_t*)(lds + L.xs);
    int16_t* s_ir = (int16_t*)(lds + L.ir);
    int16_t* s_tx = (int16_t*)(lds + L.tx);
    const int tid = threadIdx.x;
    const int b = row / a.P;
    const int j = row % a.P;
    const int S = t.S, K = t.K, m = t.m;
    const int level = a.level;
    const int NE = t.NE;
    const int64_t nb = (int64_t)b * t.NN;

    // construction weights (untempered unless asked), S1, rank by (w1 desc, id asc)
    const int cb = (level == 0) ? 1 : 1 + K + (level - 1) * NE * K;
    const int e_idx = (level == 0) ? 0 : 1 + (level - 1) * NE + j;
    const float M = key_value(s_top[0]);
    uint64_t part = 0;
    for (int i = tid; i < S; i += NT) {
        const uint64_t tk = s_top[i];
        const uint32_t w = cweight(key_value(tk), M, a.k1);
        s_w1[i] = w;
        s_k2[i] = ((uint64_t)w << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)key_id(tk));
        part += w;
    }
    const uint64_t S1 = psum<NT>(part, s_red);
    psync<NT>();
    // The support is in (logit desc, id asc) order and the weight never
    // grows along it, so ranks by (w1 desc, id asc) differ from positions
    // only where two different logits share a weight.
    bool tie = false;
    for (int i = tid + 1; i < S; i += NT)
        tie |= s_w1[i] == s_w1[i - 1] && (s_top[i] >> 32) != (s_top[i - 1] >> 32);
    if (pany<NT>(tie)) {
        rank_all<NT>(s_k2, S, s_wr);
    } else {
        for (int i = tid; i < S; i += NT) s_wr[i] = (int16_t)i;
    }
    psync<NT>();
    for (int i = tid; i < S; i += NT) s_xs[s_wr[i]] = (int16_t)i;
    psync<NT>();

    // tail q~_T (relative to x_{m+1}), its total, and its order by token id
    const float ref_t = key_value(s_top[s_xs[m]]);
    part = 0;
    for (int i = tid; i < S; i += NT) {
        const bool tail = s_wr[i] >= m;
        const uint64_t tk = s_top[i];
        const uint32_t w = tail ? cweight(key_value(tk), ref_t, a.kT) : 0u;
        s_q[i] = w;
        part += w;
        s_k2[i] = tail ? (uint64_t)(0xFFFFFFFFu - (uint32_t)key_id(tk)) + 1 : 0ull;
    }
    const uint64_t Zq = psum<NT>(part, s_red);
    psync<NT>();
    rank_all<NT>(s_k2, S, s_ir);
    psync<NT>();
    // id-sorted tail, written straight to the tree (q~ for verification)
    const int ntail = S - m;
    const int64_t tail_base = ((int64_t)b * t.E + e_idx) * S;
    for (int i = tid; i < S; i += NT) {
        if (s_wr[i] >= m) {
            const int idr = s_ir[i];
            s_tq[idr] = s_q[i];
            s_tx[idr] = (int16_t)i;
            t.tail_id[tail_base + idr] = key_id(s_top[i]);
            t.tail_q[tail_base + idr] = s_q[i];
        }
    }
    if (tid == 0) *s_yi = -1;
    psync<NT>();

    // Y ~ q~_T: t = floor(U64 Zq / 2^64), the first id-ordered tail entry
    // whose inclusive prefix exceeds t (each thread scans a contiguous block)
    const uint64_t tt = __umul64hi(u, Zq);
    const int IPT = (ntail + NT - 1) / NT;
    const int lo = min(ntail, tid * IPT), hi = min(ntail, lo + IPT);
    uint64_t mysum = 0;
    for (int i = lo; i < hi; ++i) mysum += s_tq[i];
    uint64_t acc;
    if (NT == WAVE) {
        acc = wave_incl_scan_u64(mysum) - mysum;
    } else {
        uint64_t total;
        acc = block_excl_scan_u64<NT>(mysum, s_red, &total);
    }
    if (acc <= tt && tt < acc + mysum) {
        for (int i = lo; i < hi; ++i) {
            const uint64_t w = s_tq[i];
            if (tt < acc + w) {
                *s_yi = s_tx[i];
                break;
            }
            acc += w;
        }
    }
    psync<NT>();
    int yi = *s_yi;
    if (yi < 0) {
        if (tid == 0) atomicOr(t.err, 1);
        yi = s_xs[m];                            // unreachable fallback
    }

    if (tid == 0) {
        t.zq[(int64_t)b * t.E + e_idx] = Zq;
        t.first_child[nb + pu] = cb + j * K;
        t.exp_of[nb + pu] = e_idx;
        if (level == 0) emit_root(t, nb);
    }
    // the K children: top-m leads, Y, fills (App. C.1)
    if (tid < K) {
        const int s = tid;
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
        emit_child(t, level, nb, pu, cb + j * K + s, s, kind, key_id(s_top[item]), proxy, qtrue);
    }
}

// ---------------------------------------------------------------------------
// k_pool: one block per row: parent, support (merge of the chunk lists),
// pool, and, by the last row of each sequence, the next frontier
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(NTP) void k_pool(TreeDev t, LevelArgs a) {
    extern __shared__ __align__(16) uint8_t s_pdyn[];
    __shared__ uint64_t s_red[NTP / WAVE];
    __shared__ int s_pu, s_yi;
    __shared__ uint64_t s_u;
    const PoolLds L = pool_lds(t.S, t.C);
    uint64_t* s_m = (uint64_t*)(s_pdyn + L.m);    // the C chunk lists, C * S keys
    uint64_t* s_top = (uint64_t*)(s_pdyn + L.top);
    uint64_t* s_k2 = (uint64_t*)(s_pdyn + L.k2);

    const int tid = threadIdx.x;
    const int row = blockIdx.x;
    const int b = row / a.P;
    const int j = row % a.P;
    const int S = t.S, K = t.K;
    const int C = t.C;
    const int level = a.level;
    const int NE = t.NE;
    const int64_t nb = (int64_t)b * t.NN;

    // the chunk lists, and the parent: frontier node j of the previous level
    // (the n_expand children with the highest priority, chosen by the
    // previous launch) with the Philox draw of its sampled slot
    const uint64_t* src = t.sel + (int64_t)row * C * S;
    for (int i = tid; i < C * S; i += NTP) s_m[i] = src[i];
    for (int i = tid; i < S; i += NTP) s_top[i] = 0ull;   // id -1 until merged
    if (tid == 0) {
        int pu = (level == 0) ? 0 : t.frontier[(int64_t)b * NE + j];
        const int lo_uid = (level == 0) ? 0 : ((level == 1) ? 1 : 1 + K + (level - 2) * NE * K);
        const int hi_uid = (level == 0) ? 1 : lo_uid + ((level == 1) ? 1 : NE) * K;
        if (pu < lo_uid || pu >= hi_uid) {
            atomicOr(t.err, 16);
            pu = 0;
        }
        s_pu = pu;
        s_u = (level == 0) ? philox_draw(a.rng_key, P_DRAFT, (uint64_t)b, 0ull)
                           : t.fr_u[(int64_t)b * NE + j];
        if (pu == 0 && level > 0) s_u = philox_draw(a.rng_key, P_DRAFT, (uint64_t)b, 0ull);
    }
    __syncthreads();

    // merge: a key's rank in the row is its position in its own (sorted)
    // list plus the count of larger keys in every other list (a binary
    // search per list).  Every list holds S keys (a chunk is larger than any
    // support); keys are unique and 0 marks an empty slot.  Two keys per
    // thread and four lists at a time keep eight searches in flight.
    {
        int pw2 = 1;
        while (pw2 * 2 <= S) pw2 *= 2;
        const int nk = C * S;
        for (int eA = tid; eA < nk; eA += 2 * NTP) {
            const int eB = eA + NTP;
            const uint64_t kA = s_m[eA], kB = eB < nk ? s_m[eB] : 0ull;
            const int lA = eA / S, lB = eB / S;
            int rA = eA - lA * S, rB = eB - lB * S;
            for (int c2 = 0; c2 < C; c2 += 4) {
                int oA[4] = {0, 0, 0, 0}, oB[4] = {0, 0, 0, 0};
                for (int half = pw2; half > 0; half >>= 1) {
#pragma unroll
                    for (int cc = 0; cc < 4; ++cc) {
                        if (c2 + cc < C) {
                            const uint64_t* L2 = s_m + (c2 + cc) * S;
                            const uint64_t xA = L2[min(oA[cc] + half, S) - 1];
                            const uint64_t xB = L2[min(oB[cc] + half, S) - 1];
                            oA[cc] += (oA[cc] + half <= S && xA > kA) ? half : 0;
                            oB[cc] += (oB[cc] + half <= S && xB > kB) ? half : 0;
                        }
                    }
                }
#pragma unroll
                for (int cc = 0; cc < 4; ++cc) {
                    if (c2 + cc < C && c2 + cc != lA) rA += oA[cc];
                    if (c2 + cc < C && c2 + cc != lB) rB += oB[cc];
                }
            }
            if (kA != 0ull && rA < S) s_top[rA] = kA;
            if (kB != 0ull && rB < S) s_top[rB] = kB;
        }
    }
    __syncthreads();
    for (int i = tid; i < S; i += NTP) {
        if ((uint32_t)key_id(s_top[i]) >= (uint32_t)t.V) {   // a support slot left empty
            atomicOr(t.err, 256);
            s_top[i] = logit_key(-INFINITY, 0u);
        }
    }
    __syncthreads();

    // the pool: one wave for small supports (no block barriers), else all
    if (S <= 256) {
        if (tid < WAVE) pool_form<WAVE>(t, a, row, s_pdyn, s_pu, s_u, s_red, &s_yi);
    } else {
        pool_form<NTP>(t, a, row, s_pdyn, s_pu, s_u, s_red, &s_yi);
    }
    if (level + 1 >= t.D) return;

    // the next frontier: the last row of the sequence to finish selects it
    select_frontier(t, a, b, s_top, s_k2);
}

// ---------------------------------------------------------------------------
// k_select: the exact top-Sc of one chunk of one row
// ---------------------------------------------------------------------------
template <int DT, int NVC>
__device__ __forceinline__ void select_block(const TreeDev& t, const LevelArgs& a) {
    constexpr int VEC = DT ? 8 : 4;
    constexpr int ESZ = DT ? 2 : 4;
    constexpr int NM = DT ? (NVC + 1) / 2 : NVC;   // registers of per-vector maxima

    __shared__ uint64_t s_keys[CAPC];           // candidates
    __shared__ uint4 s_cv[CAPV];                 // candidate vectors
    __shared__ int16_t s_rank[CAPC];
    __shared__ int s_cvi[CAPV];                  // their vector indices
    __shared__ uint32_t s_off[2 * NTC];          // threshold offers
    __shared__ int s_bc[2][NTC / WAVE];
    __shared__ uint32_t s_h;
    __shared__ int s_cnt, s_nv;
    __shared__ int s_redi[NTC / WAVE];

    const int tid = threadIdx.x;
    const int c = blockIdx.x;
    const int row = blockIdx.y;
    const int V = t.V;
    const int v0 = c * NTC * NVC;                           // first vector of the chunk
    const int nvalid = min(V - v0 * VEC, NTC * NVC * VEC);  // >= 1: C = ceil(V / chunk)
    const int nsel = min(t.Sc, nvalid);
    const char* base = (const char*)a.logits + (int64_t)row * t.stride * ESZ;
    uint64_t* out = t.sel + ((int64_t)row * t.C + c) * t.Sc;

    uint4 r[NVC];
#pragma unroll
    for (int i = 0; i < NVC; ++i) r[i] = load_row_vec<DT>(base, v0 + i * NTC + tid, V);
    if (tid == 0) {
        s_cnt = 0;
        s_nv = 0;
    }

    // per-vector maxima (exact) and this thread's maximum.  bf16: a packed
    // word read as fp32 is its high element plus a fraction of one bf16 ulp
    // (the low element's bits), so the maximum over the raw words and the
    // unpacked low elements, with its low 16 bits cleared, is exactly the
    // maximum element (logits and padding are finite, so no word is a NaN)
    uint32_t vm[NM];
#pragma unroll
    for (int q = 0; q < NM; ++q) vm[q] = 0;
    float tmax = -INFINITY;
#pragma unroll
    for (int i = 0; i < NVC; ++i) {
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

    // threshold tau: at least nsel elements of the chunk are >= tau.  Every
    // thread offers the 16-bit order-preserving codes of its two largest
    // vector maxima; the largest code h that nsel offered codes reach gives
    // tau = the smallest value with code h (each offered maximum is a
    // distinct vector holding an element >= tau).  One wave finds h by
    // bisection over the 2 * NTC offers.  Vectors past the row end read as
    // -inf, so tau may fall to -inf: then every element of the chunk is a
    // candidate.  Supports larger than the offers use all vector maxima.
    const int lane = tid % WAVE, wid = tid / WAVE;
    uint32_t c1 = 0, c2 = 0;
#pragma unroll
    for (int i = 0; i < NVC; ++i) {
        const float v = DT ? ((i & 1) ? bf_hi(vm[i / 2]) : bf_lo(vm[i / 2]))
                           : __uint_as_float(vm[i]);
        const uint32_t cv = ord32(v) >> 16;
        c2 = max(c2, min(c1, cv));
        c1 = max(c1, cv);
    }
    uint32_t h = 0;
    if (nsel <= 2 * NTC) {
        s_off[tid] = c1;
        s_off[NTC + tid] = c2;
        __syncthreads();
        if (wid == 0) {
            uint32_t o[2 * NTC / WAVE];
#pragma unroll
            for (int q = 0; q < 2 * NTC / WAVE; ++q) o[q] = s_off[q * WAVE + lane];
#pragma unroll 1
            for (int bit = 15; bit >= 0; --bit) {
                const uint32_t cand = h | (1u << bit);
                int n = 0;
#pragma unroll
                for (int q = 0; q < 2 * NTC / WAVE; ++q) n += __popcll(__ballot(o[q] >= cand));
                if (n >= nsel) h = cand;
            }
            if (lane == 0) s_h = h;
        }
        __syncthreads();
        h = s_h;
    } else {
#pragma unroll 1
        for (int bit = 15; bit >= 0; --bit) {
            const uint32_t cand = h | (1u << bit);
            int n = 0;
#pragma unroll
            for (int i = 0; i < NVC; ++i) {
                const float v = DT ? ((i & 1) ? bf_hi(vm[i / 2]) : bf_lo(vm[i / 2]))
                                   : __uint_as_float(vm[i]);
                n += (ord32(v) >> 16) >= cand;
            }
            n = wave_sum_i32(n);
            if (lane == 0) s_bc[bit & 1][wid] = n;
            __syncthreads();
            int tot = 0;
#pragma unroll
            for (int w = 0; w < NTC / WAVE; ++w) tot += s_bc[bit & 1][w];
            if (tot >= nsel) h = cand;
        }
    }
    const float tau = (h << 16) > ord32(-INFINITY) ? unord32(h << 16) : -INFINITY;

    // candidates >= tau in two compactions, so the per-element work touches
    // only the few vectors whose maximum reaches tau: (1) every wave counts
    // its candidate vectors with ballots, reserves LDS slots with one atomic
    // and copies them there; (2) each thread scans whole candidate vectors
    // and appends their elements >= tau the same way.
    int wn = 0;
#pragma unroll
    for (int i = 0; i < NVC; ++i) {
        const float vmax = DT ? ((i & 1) ? bf_hi(vm[i / 2]) : bf_lo(vm[i / 2]))
                              : __uint_as_float(vm[i]);
        wn += __popcll(__ballot(vmax >= tau));
    }
    int wbase = 0;
    if (lane == 0) wbase = atomicAdd(&s_nv, wn);
    wbase = (int)lane_u32((uint32_t)wbase, 0);
#pragma unroll
    for (int i = 0; i < NVC; ++i) {
        const float vmax = DT ? ((i & 1) ? bf_hi(vm[i / 2]) : bf_lo(vm[i / 2]))
                              : __uint_as_float(vm[i]);
        const bool take = vmax >= tau;
        const uint64_t msk = __ballot(take);
        if (take) {
            const int pos = wbase + (int)__builtin_amdgcn_mbcnt_hi(
                (uint32_t)(msk >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)msk, 0u));
            if (pos < CAPV) {
                s_cv[pos] = r[i];
                s_cvi[pos] = v0 + i * NTC + tid;
            }
        }
        wbase += __popcll(msk);
    }
    __syncthreads();
    const int nv = s_nv;
    if (nv <= CAPV) {
        for (int j0 = 0; j0 < nv; j0 += NTC) {
            const int j = j0 + tid;
            uint4 x = make_uint4(0, 0, 0, 0);
            int e0 = V;
            if (j < nv) {
                x = s_cv[j];
                e0 = s_cvi[j] * VEC;
            }
            int n = 0;
#pragma unroll
            for (int k = 0; k < VEC; ++k) n += (elem<DT>(x, k) >= tau) & (e0 + k < V);
            const int excl = wave_excl_scan(n);
            int base = 0;
            if (lane == WAVE - 1) base = atomicAdd(&s_cnt, excl + n);
            int pos = (int)lane_u32((uint32_t)base, WAVE - 1) + excl;
#pragma unroll
            for (int k = 0; k < VEC; ++k) {
                const float v = elem<DT>(x, k);
                if (v >= tau && e0 + k < V) {
                    if (pos < CAPC) s_keys[pos] = logit_key(v, (uint32_t)(e0 + k));
                    ++pos;
                }
            }
        }
    } else if (tid == 0) {
        s_cnt = CAPC + 1;                        // too many: exact fallback below
    }
    __syncthreads();
    int cnt = s_cnt;

    if (cnt > CAPC) {
        // Degenerate chunk (massive ties at the threshold): the nsel-th
        // largest selection key, exactly, by bisection on the 64-bit key.
        // Rare, so it re-reads the chunk from memory rather than holding more
        // registers.
        const int e_end = min(V, (v0 + NTC * NVC) * VEC);
        uint64_t x = 0;
        for (int bit = 63; bit >= 0; --bit) {
            const uint64_t cand = x | (1ull << bit);
            int n = 0;
#pragma unroll 1
            for (int i = 0; i < NVC; ++i) {
                const int vi = v0 + i * NTC + tid;
                if (vi * VEC >= e_end) continue;
                const uint4 w = load_row_vec<DT>(base, vi, V);
#pragma unroll
                for (int k = 0; k < VEC; ++k) {
                    const int id = vi * VEC + k;
                    n += (id < V) && (logit_key(elem<DT>(w, k), (uint32_t)id) >= cand);
                }
            }
            n = block_sum_i32<NTC>(n, s_redi);
            if (n >= nsel) x = cand;
        }
        __syncthreads();
        if (tid == 0) s_cnt = 0;
        __syncthreads();
#pragma unroll 1
        for (int i = 0; i < NVC; ++i) {
            const int vi = v0 + i * NTC + tid;
            if (vi * VEC >= e_end) continue;
            const uint4 w = load_row_vec<DT>(base, vi, V);
#pragma unroll
            for (int k = 0; k < VEC; ++k) {
                const int id = vi * VEC + k;
                if (id < V) {
                    const uint64_t key = logit_key(elem<DT>(w, k), (uint32_t)id);
                    if (key >= x) {
                        const int pos = atomicAdd(&s_cnt, 1);
                        if (pos < CAPC) s_keys[pos] = key;
                    }
                }
            }
        }
        __syncthreads();
        cnt = min(s_cnt, CAPC);
    }

    // exact top-nsel of the candidates, written sorted; unused slots are 0
    // (below every real key)
    rank_keys<NTC>(s_keys, cnt, s_rank);
    __syncthreads();
    for (int i = tid; i < cnt; i += NTC) {
        const int rk = s_rank[i];
        if (rk < nsel) out[rk] = s_keys[i];
    }
    for (int i = nsel + tid; i < t.Sc; i += NTC) out[i] = 0ull;

}

// Four blocks per CU keep enough loads in flight; the largest chunk variant
// holds twice the registers and runs at two.
template <int DT, int NVC>
__global__ __launch_bounds__(NTC) void k_select(TreeDev t,
                                                                                         LevelArgs a) {
    select_block<DT, NVC>(t, a);
}
template <int DT>
__global__ __launch_bounds__(NTC) void k_select_wide(TreeDev t, LevelArgs a) {
    select_block<DT, 32>(t, a);
}

// 16-byte vectors per thread of k_expand; a chunk is NTC * NVC vectors.
static const int kNVC[] = {4, 8, 16, 32};

int expand_variant_count(int) { return (int)(sizeof(kNVC) / sizeof(kNVC[0])); }

ExpandVariant expand_variant(int dtype, int v, int V, int S) {
    const int chunk = NTC * kNVC[v] * (dtype ? 8 : 4);
    ExpandVariant ev;
    ev.chunk = chunk;
    ev.C = (V + chunk - 1) / chunk;
    ev.Sc = S < chunk ? S : chunk;
    ev.ok = (int64_t)ev.C * ev.Sc <= MERGE_MAX;
    return ev;
}

template <int DT>
static void launch_dt(const TreeDev& t, const LevelArgs& a, int v, dim3 grid, size_t shm,
                      hipStream_t s) {
    switch (v) {
    case 0: k_select<DT, 4><<<grid, NTC, shm, s>>>(t, a); break;
    case 1: k_select<DT, 8><<<grid, NTC, shm, s>>>(t, a); break;
    case 2: k_select<DT, 16><<<grid, NTC, shm, s>>>(t, a); break;
    default: k_select_wide<DT><<<grid, NTC, shm, s>>>(t, a); break;
    }
}

hipError_t launch_select(const TreeDev& t, const LevelArgs& a, int variant, hipStream_t s) {
    const int rows = t.B * a.P;
    const dim3 grid(t.C, rows);
    if (t.dtype) launch_dt<1>(t, a, variant, grid, 0, s);
    else launch_dt<0>(t, a, variant, grid, 0, s);
    return hipGetLastError();
}

hipError_t launch_expand(const TreeDev& t, const LevelArgs& a, int variant, hipStream_t s) {
    hipError_t e = launch_select(t, a, variant, s);
    if (e != hipSuccess) return e;
    k_pool<<<t.B * a.P, NTP, (size_t)pool_lds(t.S, t.C).bytes, s>>>(t, a);
    return hipGetLastError();
}

int expand_variant_nvc(int v) { return kNVC[v]; }

}  // namespace rheo
