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
#include <type_traits>

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
constexpr int NTE = 512;      // threads per k_expand_row block
constexpr int EBATCH = 8;     // 16-byte vectors per thread and batch of k_expand_row
constexpr int kLargeSupport = 256;  // supports above it: the large class of k_expand_row

template <int DT>
__device__ __forceinline__ float elem(const uint4& v, int k) {
    const uint32_t* w = &v.x;
    if (DT) return (k & 1) ? bf_hi(w[k >> 1]) : bf_lo(w[k >> 1]);
    return __uint_as_float(w[k]);
}

// Vector vi (VEC consecutive elements) of a row; elements past V read as
// bf16 0xFFFF (a NaN: it drops out of the raw-word maxima below, whose
// kernels run with the IEEE mode bit clear, and its order code 0 lies below
// that of -inf) or fp32 -inf (ranked after every logit by its id).  Every
// consumer also checks the index against V.
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
            const uint32_t lo = (e0 < V) ? p16[e0] : 0xFFFFu;
            const uint32_t hi = (e0 + 1 < V) ? p16[e0 + 1] : 0xFFFFu;
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
// the pool of one row: parent, support, distributions and children
// ---------------------------------------------------------------------------
// LDS layout of the pool kernel's dynamic buffer: the chunk lists and one
// empty list after them, the support, ranking keys and per-entry
// arrays; the level's priority keys (<= 225 of them) reuse the regions of
// the support and the ranking keys.  The ranking-key region holds a power
// of two >= S keys.  top_min and
// k2_min (entries, bytes) enlarge the first two regions for callers that
// use them as scratch before the pool.
struct PoolLds {
    int m, top, k2, w1, q, wr, xs, bytes;
};
__host__ __device__ inline int pad16(int x) { return (x + 15) & ~15; }
__host__ __device__ inline int pow2_at_least(int x) {
    int p = 1;
    while (p < x) p <<= 1;
    return p;
}
__host__ __device__ inline PoolLds pool_lds(int S, int C, int top_min = 0, int k2_min = 0) {
    PoolLds L;
    int S2 = S > 256 ? S : 256;
    if (S2 < top_min) S2 = top_min;
    int k2b = 8 * pow2_at_least(S > 256 ? S : 256);
    if (k2b < k2_min) k2b = k2_min;
    L.m = 0;
    L.top = L.m + pad16(8 * (C + 1) * S);
    L.k2 = L.top + pad16(8 * S2);
    L.w1 = L.k2 + pad16(k2b);
    L.q = L.w1 + pad16(4 * S);
    L.wr = L.q + pad16(4 * S);
    L.xs = L.wr + pad16(2 * S);
    L.bytes = L.xs + pad16(2 * S);
    return L;
}

// The pool of one row from its support s_top (App. C.1), formed by NT
// threads (tid < NT).  Children fields the frontier selection reads in other
// blocks (token, score, path) are published with agent-scope atomics.
// A support slot left empty (no candidate reached it) is flagged and filled
// with a -inf key.
template <int NT>
__device__ __forceinline__ void pool_form(const TreeDev& t, const LevelArgs& a, int row,
                                          uint8_t* lds, const PoolLds& L, int pu,
                                          const ParentRec& pr, uint64_t u, uint64_t* s_red,
                                          int* s_yi) {
    uint64_t* s_top = (uint64_t*)(lds + L.top);
    uint64_t* s_k2 = (uint64_t*)(lds + L.k2);
    uint32_t* s_w1 = (uint32_t*)(lds + L.w1);
    uint32_t* s_q = (uint32_t*)(lds + L.q);
    int16_t* s_wr = (int16_t*)(lds + L.wr);
    int16_t* s_xs = (int16_t*)(lds + L.xs);
    const int tid = threadIdx.x;
    const int b = row / a.P;
    const int j = row % a.P;
    const int S = t.S, K = t.K, m = t.m;
    const int level = a.level;
    const int NE = t.NE;
    const int64_t nb = (int64_t)b * t.NN;
    const int cb = (level == 0) ? 1 : 1 + K + (level - 1) * NE * K;
    const int e_idx = (level == 0) ? 0 : 1 + (level - 1) * NE + j;
    if (tid == 0) *s_yi = -1;

    // Construction weights w1 (untempered unless asked) and, taking the rank
    // by (w1 desc, id asc) to be the support order, the tail weights of q~_T
    // relative to x_{m+1} = s_top[m], both totals in one exchange.  The
    // support is in (logit desc, id asc) order and the weight never grows
    // along it, so the rank differs from the position only where two
    // different logits share a weight: then the ranks and the tail are
    // computed again.
    //
    // The tail, x_{m+1} .. x_S in rank order, is written to the tree in that
    // order (token, q~ weight) for verification, and Y ~ q~_T is the entry
    // whose interval [mass before, mass before + q) holds
    // t = floor(U64 Zq / 2^64): the inverse CDF over the tail in rank order.
    // With at most one support entry per thread (S <= NT) the masses before
    // every entry come with the totals, from the same exchange.
    auto filled = [&](uint64_t k) {
        return (uint32_t)key_id(k) >= (uint32_t)t.V ? logit_key(-INFINITY, 0u) : k;
    };
    const float M = key_value(filled(s_top[0]));
    const float ref0 = key_value(filled(s_top[m]));
    uint64_t part1 = 0, partq = 0;
    for (int i = tid; i < S; i += NT) {
        uint64_t tk = s_top[i];
        if ((uint32_t)key_id(tk) >= (uint32_t)t.V) {   // a support slot left empty
            atomicOr(t.err, 256);
            tk = logit_key(-INFINITY, 0u);
            s_top[i] = tk;
        }
        const float v = key_value(tk);
        const uint32_t w = cweight(v, M, a.k1);
        s_w1[i] = w;
        part1 += w;
        const uint32_t q = (i >= m) ? cweight(v, ref0, a.kT) : 0u;
        s_q[i] = q;
        partq += q;
    }
    const bool one_each = S <= NT;           // thread tid holds support entry tid
    uint64_t S1, Zq, qbefore = 0;
    if (one_each) psum2_scan<NT>(part1, partq, s_red, &S1, &Zq, &qbefore);
    else psum2<NT>(part1, partq, s_red, &S1, &Zq);
    if (t.cfull) S1 = t.s1row[row];          // construction over the whole vocabulary
    if (NT == WAVE) wave_sync();             // (a block sum has synchronised)
    const int64_t tail_base = ((int64_t)b * t.E + e_idx) * S;
    bool tie = false;
    for (int i = tid + 1; i < S; i += NT)
        tie |= s_w1[i] == s_w1[i - 1] && (s_top[i] >> 32) != (s_top[i - 1] >> 32);
    // the tail and Y with the rank taken to be the position (one entry per
    // thread); the barrier of pany ends it, and tells whether two different
    // logits share a weight, which (rarely) sends everything through the
    // ranks below
    if (one_each && tid >= m && tid < S) {
        const uint32_t q = s_q[tid];
        t.tail_id[tail_base + tid - m] = key_id(s_top[tid]);
        t.tail_q[tail_base + tid - m] = q;
        const uint64_t tt = __umul64hi(u, Zq);
        if (qbefore <= tt && tt - qbefore < (uint64_t)q) *s_yi = tid;
    }
    const bool ident = !pany<NT>(tie);
    if (NT == WAVE) wave_sync();
    if (!ident) {
        for (int i = tid; i < S; i += NT)
            s_k2[i] = ((uint64_t)s_w1[i] << 32) |
                      (uint64_t)(0xFFFFFFFFu - (uint32_t)key_id(s_top[i]));
        psync<NT>();
        rank_all<NT>(s_k2, S, s_wr);
        psync<NT>();
        for (int i = tid; i < S; i += NT) s_xs[s_wr[i]] = (int16_t)i;
        psync<NT>();
        const float ref_t = key_value(s_top[s_xs[m]]);
        partq = 0;
        for (int i = tid; i < S; i += NT) {
            const uint32_t q = (s_wr[i] >= m) ? cweight(key_value(s_top[i]), ref_t, a.kT) : 0u;
            s_q[i] = q;
            partq += q;
        }
        Zq = psum<NT>(partq, s_red);
    }
    // position in the support of rank r, and rank of position i
    auto xs = [&](int r) -> int { return ident ? r : (int)s_xs[r]; };
    auto wr = [&](int i) -> int { return ident ? i : (int)s_wr[i]; };
    if (!(ident && one_each)) {
        // contiguous runs of ranks m .. S-1 per thread, a block scan of
        // their masses
        if (tid == 0) *s_yi = -1;
        const uint64_t tt = __umul64hi(u, Zq);
        const int ntail = S - m;
        const int per = (ntail + NT - 1) / NT;
        const int r0 = min(S, m + tid * per), r1 = min(S, r0 + per);
        uint64_t mine = 0;
        for (int r = r0; r < r1; ++r) mine += s_q[xs(r)];
        uint64_t tot;
        uint64_t pre = pscan_excl<NT>(mine, s_red, &tot);
        for (int r = r0; r < r1; ++r) {
            const int i = xs(r);
            const uint32_t q = s_q[i];
            t.tail_id[tail_base + r - m] = key_id(s_top[i]);
            t.tail_q[tail_base + r - m] = q;
            if (pre <= tt && tt - pre < (uint64_t)q) *s_yi = i;
            pre += q;
        }
        psync<NT>();
    }
    int yi = *s_yi;
    if (yi < 0) {
        if (tid == 0) atomicOr(t.err, 1);
        yi = xs(m);                              // unreachable fallback
    }

    if (tid == 0) {
        // q~_T is taken relative to x_{m+1}: undefined when its logit is
        // -inf (fewer than m + 1 tokens of the support above the rest)
        if (!(key_value(s_top[xs(m)]) > -INFINITY)) atomicOr(t.err, 512);
        t.zq[(int64_t)b * t.E + e_idx] = Zq;
        t.first_child[nb + pu] = cb + j * K;
        t.exp_of[nb + pu] = e_idx;
        if (level == 0) emit_root(t, nb);
    }
    // the K children: top-m leads, Y, fills (App. C.1); pure top-K pools:
    // the K best by (w1 desc, id asc)
    if (tid < K) {
        const int s = tid;
        const int yr = wr(yi);
        int item, kind;
        if (t.topk) {
            item = xs(s);
            kind = LEAD;
        } else if (s < m) {
            item = xs(s);
            kind = LEAD;
        } else if (s == m) {
            item = yi;
            kind = SAMPLED;
        } else {
            const int f = s - m - 1;
            const int rk = m + f + ((m + f) >= yr ? 1 : 0);
            item = xs(rk);
            kind = FILL;
        }
        double proxy;
        const double dS1 = (double)S1;
        if (kind == SAMPLED) {
            if (m >= 1) {
                uint64_t lead = 0;
                for (int q2 = 0; q2 < m; ++q2) lead += s_w1[xs(q2)];
                const uint64_t z = S1 - lead;
                const uint64_t wm = s_w1[xs(m - 1)];
                proxy = __ddiv_rn((double)(wm < z ? wm : z), dS1);
            } else {
                proxy = fmin(1.0, __dadd_rn(__ddiv_rn((double)s_w1[xs(0)], dS1), t.eps));
            }
        } else {
            proxy = __ddiv_rn((double)s_w1[item], dS1);
        }
        const double qtrue = (kind == SAMPLED) ? __ddiv_rn((double)s_q[item], (double)Zq) : proxy;
        emit_child(t, level, nb, pu, pr, cb + j * K + s, s, kind, key_id(s_top[item]), proxy,
                   qtrue,
                   wr(item) >= m ? wr(item) - m : -1);
    }
}

// The parent of row j of sequence b: frontier node j of the previous level
// (the n_expand children with the highest priority, chosen by the previous
// launch), with the Philox draw of its sampled slot (keyed by that launch's
// rng_key and the parent's uid).  One thread.  The load is issued by
// row_parent_load, the draw may be taken early (has_u), and row_parent
// checks both, so a kernel can do this work while it streams its row.
struct RowParentRaw {
    int pu;
    uint64_t u;
};
__device__ __forceinline__ RowParentRaw row_parent_load(const TreeDev& t, const LevelArgs& a,
                                                        int b, int j) {
    RowParentRaw r{0, 0ull};
    if (a.level > 0) r.pu = t.frontier[(int64_t)b * t.NE + j];
    return r;
}
__device__ __forceinline__ uint64_t parent_draw(const LevelArgs& a, int b, int pu) {
    return philox_draw(a.fr_key, P_DRAFT, (uint64_t)b, (uint64_t)pu);
}
__device__ __forceinline__ void row_parent(const TreeDev& t, const LevelArgs& a, int b, int j,
                                           const RowParentRaw& raw, bool has_u, int* s_pu,
                                           uint64_t* s_u) {
    const int level = a.level, K = t.K, NE = t.NE;
    int pu = raw.pu;
    const int lo_uid = (level == 0) ? 0 : ((level == 1) ? 1 : 1 + K + (level - 2) * NE * K);
    const int hi_uid = (level == 0) ? 1 : lo_uid + ((level == 1) ? 1 : NE) * K;
    if (pu < lo_uid || pu >= hi_uid) {
        atomicOr(t.err, 16);
        pu = 0;
    }
    *s_pu = pu;
    // the root (level 0, or the fallback above) is drawn with this launch's key
    *s_u = (pu == 0) ? philox_draw(a.rng_key, P_DRAFT, (uint64_t)b, 0ull)
                     : (has_u ? raw.u : parent_draw(a, b, pu));
}

// ---------------------------------------------------------------------------
// k_pool: one block per row: parent, support (merge of the chunk lists),
// pool, and, by the last row of each sequence, the next frontier
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(NTP) void k_pool(TreeDev t, LevelArgs a) {
    extern __shared__ __align__(16) uint8_t s_pdyn[];
    __shared__ uint64_t s_red[2 * NTP / WAVE];
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

    // the parent: frontier node j of the previous level (the n_expand
    // children with the highest priority, chosen by the previous launch)
    // with the Philox draw of its sampled slot; and the chunk lists, with
    // an empty list after them
    const int C4 = (C + 3) & ~3;
    if (tid == 0) row_parent(t, a, b, j, row_parent_load(t, a, b, j), false, &s_pu, &s_u);
    const uint64_t* src = t.sel + (int64_t)row * C * S;
    for (int i = tid; i < C * S; i += NTP) s_m[i] = src[i];
    for (int i = C * S + tid; i < (C + 1) * S; i += NTP) s_m[i] = 0ull;
    for (int i = tid; i < S; i += NTP) s_top[i] = 0ull;   // id -1 until merged
    __syncthreads();
    // the parent record, for the children written at the end
    const ParentRec pr = (tid < K) ? parent_rec(t, level, nb, s_pu) : ParentRec{1.0, 0ull};

    // merge: a key's rank in the row is its position in its own (sorted)
    // list plus the count of larger keys in every other list (a binary
    // search per list).  Every list holds S keys (a chunk is larger than any
    // support); keys are unique and 0 marks an empty slot.  Two keys per
    // thread and four lists at a time (the empty list stands in for lists
    // past the last), with no branches, keep eight loads in flight per
    // search step.
    {
        int pw2 = 1;
        while (pw2 * 2 <= S) pw2 *= 2;
        const int nk = C * S;
        for (int eA = tid; eA < nk; eA += 2 * NTP) {
            const int eB = eA + NTP;
            const uint64_t kA = s_m[eA], kB = eB < nk ? s_m[eB] : 0ull;
            const int lA = eA / S, lB = eB / S;
            int rA = eA - lA * S, rB = eB - lB * S;
            for (int c2 = 0; c2 < C4; c2 += 4) {
                int lb[4];
#pragma unroll
                for (int cc = 0; cc < 4; ++cc) lb[cc] = min(c2 + cc, C) * S;
                int oA[4] = {0, 0, 0, 0}, oB[4] = {0, 0, 0, 0};
                for (int half = pw2; half > 0; half >>= 1) {
                    uint64_t xA[4], xB[4];
#pragma unroll
                    for (int cc = 0; cc < 4; ++cc) {
                        xA[cc] = s_m[lb[cc] + min(oA[cc] + half, S) - 1];
                        xB[cc] = s_m[lb[cc] + min(oB[cc] + half, S) - 1];
                    }
#pragma unroll
                    for (int cc = 0; cc < 4; ++cc) {
                        oA[cc] += (oA[cc] + half <= S && xA[cc] > kA) ? half : 0;
                        oB[cc] += (oB[cc] + half <= S && xB[cc] > kB) ? half : 0;
                    }
                }
#pragma unroll
                for (int cc = 0; cc < 4; ++cc) {
                    rA += (c2 + cc != lA) ? oA[cc] : 0;
                    rB += (c2 + cc != lB) ? oB[cc] : 0;
                }
            }
            if (kA != 0ull && rA < S) s_top[rA] = kA;
            if (kB != 0ull && rB < S) s_top[rB] = kB;
        }
    }
    __syncthreads();

    // the pool, formed by the whole block
    pool_form<NTP>(t, a, row, s_pdyn, L, s_pu, pr, s_u, s_red, &s_yi);
    if (level + 1 >= t.D) return;

    // the next frontier: the last row of the sequence to finish selects it
    select_frontier(t, a, b, s_top, s_k2);
}

// ---------------------------------------------------------------------------
// k_select: the exact top-Sc of one chunk of one row
// ---------------------------------------------------------------------------
// A bf16 chunk holds at most 65536 elements, so its candidates are ranked by
// 32-bit keys: the 16-bit order code of the value above the complement of
// the chunk-local index (larger key = larger logit, then smaller id).  fp32
// chunks use the 64-bit row keys.
__device__ __forceinline__ uint32_t chunk_key32(float v, int lid) {
    return (ord32(v) & 0xFFFF0000u) | (uint32_t)(0xFFFF - lid);
}
// The row key (logit_key) of a chunk key; e0 = the chunk's first element.
__device__ __forceinline__ uint64_t row_key_of32(uint32_t k, int e0) {
    const uint32_t o = (k & 0xFFFF0000u) | ((k & 0x80000000u) ? 0u : 0xFFFFu);
    const uint32_t id = (uint32_t)(e0 + 0xFFFF - (int)(k & 0xFFFFu));
    return ((uint64_t)o << 32) | (uint64_t)(0xFFFFFFFFu - id);
}

// max(a, b, c) in one instruction; with the IEEE mode bit clear (the
// caller's kernel runs ieee_mode_off first) a NaN operand is ignored.
// Volatile: kept in program order after the mode change.
__device__ __forceinline__ float max3_nan_drop(float a, float b, float c) {
    float r;
    asm volatile("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
    return r;
}

// Exact maximum element of a vector of eight bf16 (raw word bits: a packed
// word read as fp32 is its high element plus a fraction of one bf16 ulp made
// of the low element's bits, so the maximum over the raw words and the
// unpacked low elements, with its low 16 bits cleared, is exactly the
// largest element).  A word whose high element is -inf (and low element not
// +0) is a NaN and is dropped, which loses nothing: -inf is the least
// logit, and the low element counts through its own unpacked operand.
// Padding (0xFFFF) drops out the same way; a vector of padding alone gives
// a NaN (order code 0).  Returned with garbage in the low 16 bits.
__device__ __forceinline__ uint32_t bf16x8_max_raw(const uint4& v) {
    float m = max3_nan_drop(__uint_as_float(v.x), bf_lo(v.x), __uint_as_float(v.y));
    m = max3_nan_drop(m, bf_lo(v.y), __uint_as_float(v.z));
    m = max3_nan_drop(m, bf_lo(v.z), __uint_as_float(v.w));
    m = max3_nan_drop(m, bf_lo(v.w), bf_lo(v.w));
    return __float_as_uint(m);
}

typedef short rs_short2 __attribute__((ext_vector_type(2)));
typedef unsigned short rs_ushort2 __attribute__((ext_vector_type(2)));
// Order codes of two packed bf16 values (negative: all bits flipped,
// otherwise the sign bit set), two lanes of 16 bits at once.
__device__ __forceinline__ rs_ushort2 bf16x2_codes(uint32_t w) {
    const rs_short2 s = __builtin_bit_cast(rs_short2, w);
    const uint32_t m = __builtin_bit_cast(uint32_t, (rs_short2)(s >> (short)15)) | 0x80008000u;
    return __builtin_bit_cast(rs_ushort2, w ^ m);
}

template <int NT>
__device__ void rank_keys32(const uint32_t* keys, int n, int16_t* rank) {
    int npad = 1;
    while (npad < n) npad <<= 1;
    int F = NT / npad;
    if (F < 1) F = 1;
    if (F > WAVE) F = WAVE;
    const int sub = threadIdx.x % F;
    const int per = NT / F;
    const uint4* k4 = (const uint4*)keys;
    const int n4 = n >> 2;
    for (int base = 0; base < n; base += per) {
        const int i = base + threadIdx.x / F;
        int cnt = 0;
        if (i < n) {
            const uint32_t k = keys[i];
#pragma unroll 4
            for (int g = sub; g < n4; g += F) {
                const uint4 x = k4[g];
                cnt += (int)(x.x > k) + (int)(x.y > k) + (int)(x.z > k) + (int)(x.w > k);
            }
            for (int j = 4 * n4 + sub; j < n; j += F) cnt += (int)(keys[j] > k);
        }
        for (int o = 1; o < F; o <<= 1) cnt += __shfl_xor(cnt, o);
        if (i < n && sub == 0) rank[i] = (int16_t)cnt;
    }
}

// Lane l (a constant) of v replaced by the wave-uniform s.
__device__ __forceinline__ int writelane_i32(int v, int s, int l) {
    asm volatile("v_writelane_b32 %0, %1, %2" : "+v"(v) : "s"(s), "n"(l));
    return v;
}

// h = the largest 16-bit code that at least nsel of the offered codes reach
// (c1 and c2 of every thread, and c3 and c4 too if `four`, a block-uniform
// flag), four bits per round: each wave counts its offers >= h | d << sh
// for d = 1..15 with ballots, lane d of the wave stores that count, the
// waves' counts are added, and d is the largest one whose count still
// reaches nsel.  s_cnt holds 2 * (NT / WAVE) * 16 ints.  Needs nsel <= the
// number of offers; all threads of the block call it.
template <int NT>
__device__ __forceinline__ uint32_t offer_threshold(uint32_t c1, uint32_t c2, uint32_t c3,
                                                    uint32_t c4, bool four, int nsel,
                                                    int* s_cnt) {
    constexpr int NW = NT / WAVE;
    const int lane = threadIdx.x % WAVE, wid = threadIdx.x / WAVE;
    uint32_t h = 0;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int sh = 12 - 4 * r;
        int* buf = s_cnt + (r & 1) * NW * 16;
        // h has no bits at or below this digit, so c >= h | d << sh is
        // ((c - h, saturated at 0) >> sh) >= d: a compare with a small constant
        const uint32_t e1 = __builtin_elementwise_sub_sat(c1, h) >> sh;
        const uint32_t e2 = __builtin_elementwise_sub_sat(c2, h) >> sh;
        const uint32_t e3 = __builtin_elementwise_sub_sat(c3, h) >> sh;
        const uint32_t e4 = __builtin_elementwise_sub_sat(c4, h) >> sh;
        int mine = 0;
        if (four) {
#pragma unroll
            for (int d = 1; d < 16; ++d) {
                const uint32_t cd = (uint32_t)d;
                const int n = __popcll(__ballot(e1 >= cd)) + __popcll(__ballot(e2 >= cd)) +
                              __popcll(__ballot(e3 >= cd)) + __popcll(__ballot(e4 >= cd));
                mine = writelane_i32(mine, n, d);
            }
        } else {
#pragma unroll
            for (int d = 1; d < 16; ++d) {
                const uint32_t cd = (uint32_t)d;
                const int n = __popcll(__ballot(e1 >= cd)) + __popcll(__ballot(e2 >= cd));
                mine = writelane_i32(mine, n, d);
            }
        }
        if (lane < 16) buf[wid * 16 + lane] = mine;
        __syncthreads();
        int tot = 0;
        if (lane < 16) {
#pragma unroll
            for (int w = 0; w < NW; ++w) tot += buf[w * 16 + lane];
        }
        const uint64_t ok = __ballot(lane >= 1 && lane < 16 && tot >= nsel);
        const uint32_t d = ok ? (uint32_t)(63 - __builtin_clzll(ok)) : 0u;
        h |= d << sh;
    }
    return h;
}
template <int NT>
__device__ __forceinline__ uint32_t offer_threshold(uint32_t c1, uint32_t c2, int nsel,
                                                    int* s_cnt) {
    return offer_threshold<NT>(c1, c2, 0u, 0u, false, nsel, s_cnt);
}

// The largest bin b of a 256-bin histogram in LDS whose suffix count (bins
// >= b) reaches need, and the count of the bins above it (.y); (-1, 0) if
// none does.  Threads 0..255 hold one bin each; s_w holds 9 ints.  All
// threads of the block call it; it ends with a barrier.
template <int NT>
__device__ __forceinline__ int2 suffix_pick256(const int* hist, int need, int* s_w) {
    static_assert(NT >= 256, "one bin per thread");
    const int t = threadIdx.x, lane = t % WAVE, w = t / WAVE;
    const int v = (t < 256) ? hist[t] : 0;
    const int ex = wave_excl_scan(v);
    const int wt = (int)lane_u32((uint32_t)(ex + v), WAVE - 1);
    if (t < 256 && lane == 0) s_w[w] = wt;
    __syncthreads();
    int higher = 0;
    if (t < 256) {
        for (int x = w + 1; x < 256 / WAVE; ++x) higher += s_w[x];
    }
    const int suf = wt - ex + higher;               // sum of bins >= t
    const uint64_t ok = __ballot(t < 256 && suf >= need);
    const int top = ok ? w * WAVE + 63 - __builtin_clzll(ok) : -1;
    if (t < 256 && lane == 0) s_w[4 + w] = top;
    __syncthreads();
    const int bin = max(max(s_w[4], s_w[5]), max(s_w[6], s_w[7]));
    if (t == bin) s_w[8] = suf - v;
    __syncthreads();
    return make_int2(bin, bin >= 0 ? s_w[8] : 0);
}

// Exact selection for a degenerate range: more candidates than LDS holds
// (massive ties at the threshold, or large values crowded into few
// threads).  The range is NQ vectors per thread, vector q of this thread at
// index vfirst + q * NT + tid; elements at V and beyond do not count;
// push(v, id) records an element.  Rare, so it re-reads the range, four
// vectors at a time.  bf16: count the elements whose code lies above the
// threshold code h; if the nsel-th largest element has code h, take
// everything above h and the smallest ids among those at h (ranks of the
// ties in id order from per-wave counts and wave scans); if it lies above h
// and the elements above h fit (at most cap), take those.  Otherwise, and for
// fp32, find the nsel-th largest key by bisection.  Ends with a barrier.
template <int DT, int NT, int NQ, typename Push>
__device__ void exact_select_fallback(const char* base, int V, int vfirst, uint32_t h, int nsel,
                                      int cap, Push push, int* s_redi,
                                      int (*s_tie)[NT / WAVE]) {
    constexpr int VEC = DT ? 8 : 4;
    constexpr int NW = NT / WAVE;
    static_assert(NQ % 4 == 0 && NQ <= 64, "re-read in groups of four vectors");
    const int tid = threadIdx.x, lane = tid % WAVE, wid = tid / WAVE;
    // an opaque trip count keeps each pass a loop (re-reading per pass)
    // rather than one straight-line block holding every element
    int nq = NQ;
    asm volatile("" : "+s"(nq));
    auto group = [&](int q0, uint4 (&w)[4]) {
        // an opaque index keeps every pass's loads (and what is computed
        // from them) inside its loop instead of live across the passes
        int vf = vfirst;
        asm volatile("" : "+v"(vf));
#pragma unroll
        for (int q = 0; q < 4; ++q) w[q] = load_row_vec<DT>(base, vf + (q0 + q) * NT + tid, V);
    };
    bool done = false;
    if (DT) {
        int ngt = 0;
#pragma unroll 1
        for (int q0 = 0; q0 < nq; q0 += 4) {
            uint4 w[4];
            group(q0, w);
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int e0 = (vfirst + (q0 + q) * NT + tid) * VEC;
#pragma unroll
                for (int k = 0; k < VEC; ++k)
                    ngt += (e0 + k < V && (ord32(elem<DT>(w[q], k)) >> 16) > h) ? 1 : 0;
            }
        }
        ngt = block_sum_i32<NT>(ngt, s_redi);
        if (ngt < nsel) {
            // ties at h, in id order: vector q, then thread, then element
            const int need = nsel - ngt;
#pragma unroll 1
            for (int q0 = 0; q0 < nq; q0 += 4) {
                uint4 w[4];
                group(q0, w);
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int e0 = (vfirst + (q0 + q) * NT + tid) * VEC;
                    int nt = 0;
#pragma unroll
                    for (int k = 0; k < VEC; ++k)
                        nt += (e0 + k < V && (ord32(elem<DT>(w[q], k)) >> 16) == h) ? 1 : 0;
                    const int tot = wave_sum_i32(nt);
                    if (lane == 0) s_tie[q0 + q][wid] = tot;
                }
            }
            __syncthreads();
            int prior = 0;                   // ties in the vectors before q, all threads
#pragma unroll 1
            for (int q0 = 0; q0 < nq; q0 += 4) {
                uint4 w[4];
                group(q0, w);
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int e0 = (vfirst + (q0 + q) * NT + tid) * VEC;
                    int nt = 0;
#pragma unroll
                    for (int k = 0; k < VEC; ++k)
                        nt += (e0 + k < V && (ord32(elem<DT>(w[q], k)) >> 16) == h) ? 1 : 0;
                    int rk = prior + wave_excl_scan(nt);
#pragma unroll
                    for (int ww = 0; ww < NW; ++ww) {
                        rk += (ww < wid) ? s_tie[q0 + q][ww] : 0;
                        prior += s_tie[q0 + q][ww];
                    }
#pragma unroll
                    for (int k = 0; k < VEC; ++k) {
                        const float v = elem<DT>(w[q], k);
                        const uint32_t cd = ord32(v) >> 16;
                        if (e0 + k < V) {
                            if (cd > h) {
                                push(v, e0 + k);
                            } else if (cd == h) {
                                if (rk < need) push(v, e0 + k);
                                ++rk;
                            }
                        }
                    }
                }
            }
            done = true;
        } else if (ngt <= cap) {
#pragma unroll 1
            for (int q0 = 0; q0 < nq; q0 += 4) {
                uint4 w[4];
                group(q0, w);
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int e0 = (vfirst + (q0 + q) * NT + tid) * VEC;
#pragma unroll
                    for (int k = 0; k < VEC; ++k) {
                        const float v = elem<DT>(w[q], k);
                        if (e0 + k < V && (ord32(v) >> 16) > h) push(v, e0 + k);
                    }
                }
            }
            done = true;
        }
    }
    if (!done) {
        uint64_t x = 0;
#pragma unroll 1
        for (int bit = 63; bit >= 0; --bit) {
            const uint64_t cand = x | (1ull << bit);
            int n = 0;
#pragma unroll 1
            for (int q0 = 0; q0 < nq; q0 += 4) {
                uint4 w[4];
                group(q0, w);
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int e0 = (vfirst + (q0 + q) * NT + tid) * VEC;
#pragma unroll
                    for (int k = 0; k < VEC; ++k)
                        n += (e0 + k < V &&
                              logit_key(elem<DT>(w[q], k), (uint32_t)(e0 + k)) >= cand) ? 1 : 0;
                }
            }
            n = block_sum_i32<NT>(n, s_redi);
            if (n >= nsel) x = cand;
        }
#pragma unroll 1
        for (int q0 = 0; q0 < nq; q0 += 4) {
            uint4 w[4];
            group(q0, w);
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int e0 = (vfirst + (q0 + q) * NT + tid) * VEC;
#pragma unroll
                for (int k = 0; k < VEC; ++k) {
                    const float v = elem<DT>(w[q], k);
                    if (e0 + k < V && logit_key(v, (uint32_t)(e0 + k)) >= x) push(v, e0 + k);
                }
            }
        }
    }
    __syncthreads();
}

// The candidate count after exact_select_fallback (which ends with a
// barrier): an atomic load behind a compiler barrier, since the call is not
// inlined and a plain load of the counter may be scheduled before it.
__device__ __forceinline__ int fallback_count(int* cnt) {
    asm volatile("" ::: "memory");
    return __hip_atomic_load(cnt, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

template <int DT, int NVC>
__device__ __forceinline__ void select_block(const TreeDev& t, const LevelArgs& a) {
    constexpr int VEC = DT ? 8 : 4;
    constexpr int NM = DT ? (NVC + 1) / 2 : NVC;   // registers of per-vector maxima
    constexpr int NW = NTC / WAVE;
    constexpr int WCAP = CAPV / NW;                // candidate vectors per wave

    __shared__ __align__(16) uint64_t s_keys[CAPC];   // candidates (bf16: 32-bit keys)
    __shared__ uint4 s_cv[CAPV];                 // candidate vectors, WCAP per wave
    __shared__ int16_t s_rank[CAPC];
    __shared__ int s_cvi[CAPV];                  // their vector indices
    __shared__ int s_thr[2 * NW * 16];          // threshold counts
    __shared__ int s_bc[2][NW];
    __shared__ int s_wn[NW];
    __shared__ int s_cnt;
    __shared__ int s_redi[NW];
    uint32_t* s_k32 = (uint32_t*)s_keys;

    ieee_mode_off();                             // NaN words drop out of the maxima
    const int tid = threadIdx.x;
    const int lane = tid % WAVE, wid = tid / WAVE;
    const int c = blockIdx.x;
    const int row = blockIdx.y;
    const int V = t.V;
    const int v0 = c * NTC * NVC;                           // first vector of the chunk
    const int nvalid = min(V - v0 * VEC, NTC * NVC * VEC);  // >= 1: C = ceil(V / chunk)
    const int nsel = min(t.Sc, nvalid);
    const int NVR = (V + VEC - 1) / VEC;                    // vectors of the row
    const char* base = (const char*)a.logits + (int64_t)row * t.stride * (DT ? 2 : 4);
    uint64_t* out = t.sel + ((int64_t)row * t.C + c) * t.Sc;

    // the chunk, NVC 16-byte vectors per thread; every chunk but a row's
    // last is whole, so its loads need no bounds checks
    uint4 r[NVC];
    if ((v0 + NTC * NVC) * VEC <= V) {
        const uint32_t toff = (uint32_t)tid * 16u;
#pragma unroll
        for (int i = 0; i < NVC; ++i)
            r[i] = load_stream16(base + (int64_t)(v0 + i * NTC) * 16 + toff);
    } else {
#pragma unroll
        for (int i = 0; i < NVC; ++i) r[i] = load_row_vec<DT>(base, v0 + i * NTC + tid, V);
    }
    if (tid == 0) s_cnt = 0;

    // per-vector maxima (exact; bf16: two per register, high halves) and
    // every thread's two largest as 16-bit order codes
    uint32_t vm[NM];
    uint32_t c1 = 0, c2 = 0;
    if (DT) {
        rs_ushort2 p1 = {0, 0}, p2 = {0, 0};
#pragma unroll
        for (int q = 0; q < NM; ++q) {
            const uint32_t lo = bf16x8_max_raw(r[2 * q]);
            const uint32_t hi = (2 * q + 1 < NVC) ? bf16x8_max_raw(r[2 * q + 1]) : lo;
            vm[q] = __builtin_amdgcn_perm(hi, lo, 0x07060302u);
            const rs_ushort2 cq = bf16x2_codes(vm[q]);
            p2 = __builtin_elementwise_max(p2, __builtin_elementwise_min(p1, cq));
            p1 = __builtin_elementwise_max(p1, cq);
        }
        c1 = max((uint32_t)p1.x, (uint32_t)p1.y);
        c2 = max(min((uint32_t)p1.x, (uint32_t)p1.y), max((uint32_t)p2.x, (uint32_t)p2.y));
    } else {
#pragma unroll
        for (int i = 0; i < NVC; ++i) {
            const float mx = fmaxf(fmaxf(elem<DT>(r[i], 0), elem<DT>(r[i], 1)),
                                   fmaxf(elem<DT>(r[i], 2), elem<DT>(r[i], 3)));
            vm[i] = __float_as_uint(mx);
            const uint32_t cv = ord32(mx) >> 16;
            c2 = max(c2, min(c1, cv));
            c1 = max(c1, cv);
        }
    }

    // threshold tau: at least nsel elements of the chunk are >= tau.  Every
    // thread offers the order codes of its two largest vector maxima; h =
    // the nsel-th largest offered code gives tau = the smallest value with
    // code h (each offered maximum is a distinct vector holding an element
    // >= tau), found four bits at a time (offer_threshold).  Elements past
    // the row end read as -inf (fp32) or a NaN word (bf16), so in a row's
    // last chunk tau may fall to -inf; vectors wholly past the row end are
    // never candidates, so the candidates are then the chunk's valid
    // elements.  Supports larger than the offers use all vector maxima.
    static_assert(NTC == 256, "one histogram bin per thread");
    uint32_t h = 0;
    if (nsel <= 2 * NTC) {
        h = offer_threshold<NTC>(c1, c2, nsel, s_thr);
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
            for (int w = 0; w < NW; ++w) tot += s_bc[bit & 1][w];
            if (tot >= nsel) h = cand;
        }
    }
    const float tau = (h << 16) > ord32(-INFINITY) ? unord32(h << 16) : -INFINITY;

    // candidates >= tau in two compactions, so the per-element work touches
    // only the few vectors whose maximum reaches tau: (1) every wave appends
    // its candidate vectors to its own LDS region (ballot and bit count);
    // (2) the threads take the candidate vectors of all regions in turn and
    // append their elements >= tau to the candidate list.  If a wave has more
    // candidate vectors than its region holds, but all fit, they are written
    // again into one list with slots reserved per wave; more than that sends
    // the chunk to the exact fallback below.
    {
        int wpos = 0;
#pragma unroll
        for (int i = 0; i < NVC; ++i) {
            const float vmax = DT ? ((i & 1) ? bf_hi(vm[i / 2]) : bf_lo(vm[i / 2]))
                                  : __uint_as_float(vm[i]);
            const bool take = vmax >= tau && v0 + i * NTC + tid < NVR;
            const uint64_t msk = __ballot(take);
            if (take) {
                const int pos = wpos + (int)__builtin_amdgcn_mbcnt_hi(
                    (uint32_t)(msk >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)msk, 0u));
                if (pos < WCAP) {
                    s_cv[wid * WCAP + pos] = r[i];
                    s_cvi[wid * WCAP + pos] = v0 + i * NTC + tid;
                }
            }
            wpos += __popcll(msk);
        }
        if (lane == 0) s_wn[wid] = wpos;
    }
    __syncthreads();
    int wn[NW], nv = 0, wbefore = 0;
    bool ovf = false;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
        wn[w] = s_wn[w];
        ovf |= wn[w] > WCAP;
        wbefore += (w < wid) ? wn[w] : 0;
        nv += wn[w];
    }
    const bool contig = ovf && nv <= CAPV;
    if (contig) {
        // one list: each wave's vectors after those of the waves before it
        int wpos = wbefore;
#pragma unroll
        for (int i = 0; i < NVC; ++i) {
            const float vmax = DT ? ((i & 1) ? bf_hi(vm[i / 2]) : bf_lo(vm[i / 2]))
                                  : __uint_as_float(vm[i]);
            const bool take = vmax >= tau && v0 + i * NTC + tid < NVR;
            const uint64_t msk = __ballot(take);
            if (take) {
                const int pos = wpos + (int)__builtin_amdgcn_mbcnt_hi(
                    (uint32_t)(msk >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)msk, 0u));
                s_cv[pos] = r[i];
                s_cvi[pos] = v0 + i * NTC + tid;
            }
            wpos += __popcll(msk);
        }
        __syncthreads();
    }
    if (!ovf || contig) {
        for (int j0 = 0; j0 < nv; j0 += NTC) {
            const int j = j0 + tid;
            // entry j of the concatenated regions (or of the one list)
            int w = 0, off = j;
            if (!contig) {
#pragma unroll
                for (int q = 0; q < NW - 1; ++q) {
                    const bool past = off >= wn[q] && w == q;
                    off -= past ? wn[q] : 0;
                    w += past ? 1 : 0;
                }
            }
            uint4 x = make_uint4(0, 0, 0, 0);
            int e0 = V;
            if (j < nv) {
                x = s_cv[w * WCAP + off];
                e0 = s_cvi[w * WCAP + off] * VEC;
            }
            int n = 0;
#pragma unroll
            for (int k = 0; k < VEC; ++k) n += (elem<DT>(x, k) >= tau) & (e0 + k < V);
            const int excl = wave_excl_scan(n);
            int cbase = 0;
            if (lane == WAVE - 1) cbase = atomicAdd(&s_cnt, excl + n);
            int pos = (int)lane_u32((uint32_t)cbase, WAVE - 1) + excl;
#pragma unroll
            for (int k = 0; k < VEC; ++k) {
                const float v = elem<DT>(x, k);
                if (v >= tau && e0 + k < V) {
                    if (pos < CAPC) {
                        if (DT) s_k32[pos] = chunk_key32(v, e0 + k - v0 * VEC);
                        else s_keys[pos] = logit_key(v, (uint32_t)(e0 + k));
                    }
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
        // degenerate chunk: exact selection from the chunk in memory
        const int eb = v0 * VEC;                 // first element of the chunk
        __shared__ int s_tie[32][NW];
        __syncthreads();
        if (tid == 0) s_cnt = 0;
        exact_select_fallback<DT, NTC, NVC>(
            base, V, v0, h, nsel, CAPC,
            [&](float v, int id) {
                const int pos = atomicAdd(&s_cnt, 1);
                if (pos < CAPC) {
                    if (DT) s_k32[pos] = chunk_key32(v, id - eb);
                    else s_keys[pos] = logit_key(v, (uint32_t)id);
                }
            },
            s_redi, s_tie);
        cnt = min(fallback_count(&s_cnt), CAPC);
    }

    // exact top-nsel of the candidates, written sorted; unused slots are 0
    // (below every real key)
    if (DT) rank_keys32<NTC>(s_k32, cnt, s_rank);
    else rank_keys<NTC>(s_keys, cnt, s_rank);
    __syncthreads();
    for (int i = tid; i < cnt; i += NTC) {
        const int rk = s_rank[i];
        if (rk < nsel) out[rk] = DT ? row_key_of32(s_k32[i], v0 * VEC) : s_keys[i];
    }
    for (int i = nsel + tid; i < t.Sc; i += NTC) out[i] = 0ull;
}


// ---------------------------------------------------------------------------
// k_expand_row: the whole level for one row per block.  The row is streamed
// once (double-buffered batches of 16-byte vectors; only each vector's
// exact maximum is kept, as a 16-bit order code in registers); the
// threshold comes from the largest vector maxima every thread offers (two,
// or four for supports above 128), and for supports above kLargeSupport
// (LS) is raised to the exact S-th largest vector maximum by two rounds of
// a 256-bin histogram; only the candidate vectors are read again; their
// elements at or above the threshold are ranked (LS: sorted) into the
// support, then the pool (App. C.1) and, by the last row of each sequence,
// the next frontier -- with no chunk lists, no merge and no second launch.
// Used when the row fits NQ vectors per thread and the level has enough
// rows to fill the chip.
// ---------------------------------------------------------------------------
constexpr int CAPV_L = 2048;  // candidate vectors of a large-support row
constexpr int CAPC_L = 2048;  // candidates of a large-support row (sorted in place)

// Dynamic LDS of k_expand_row: the pool layout; large supports sort their
// candidates in the support region and list candidate vectors in the
// ranking-key region, both free until the pool is formed.
__host__ __device__ inline PoolLds row_lds(int S, bool ls) {
    return ls ? pool_lds(S, 0, CAPC_L, 4 * CAPV_L) : pool_lds(S, 0);
}

// SC: the support class -- 0: S <= 128 (two offers per thread), 1: S <= 256
// (four offers), 2: larger supports (LS).
template <int DT, int NQ, int SC, int NTB>
__global__ __launch_bounds__(NTB) void k_expand_row(TreeDev t, LevelArgs a) {
    constexpr bool LS = SC == 2;
    constexpr bool four = SC >= 1;
    constexpr int VEC = DT ? 8 : 4;
    constexpr int NW = NTB / WAVE;
    constexpr int NB = NQ / EBATCH;
    constexpr int NM = DT ? NQ / 2 : NQ;
    constexpr int CV = LS ? CAPV_L : CAPV;      // candidate vectors held
    constexpr int CC = LS ? CAPC_L : CAPC;      // candidates held
    static_assert(NQ % (2 * EBATCH) == 0 && NQ <= 64, "batches come in pairs");
    // candidate-vector masks: bf16 vector 2 qi at bit qi, 2 qi + 1 at bit
    // HALF + qi; fp32 vector q at bit q
    using mask_t = typename std::conditional<(NQ > 32), uint64_t, uint32_t>::type;
    constexpr int HALF = NQ > 32 ? 32 : 16;
    extern __shared__ __align__(16) uint8_t s_pdyn[];
    __shared__ __align__(16) uint64_t s_keys_st[LS ? 2 : CAPC];
    __shared__ int16_t s_rank[LS ? 2 : CAPC];
    __shared__ int s_cvi_st[LS ? 1 : CAPV];
    __shared__ int s_hist[LS ? 256 : 1];
    __shared__ int s_thr[2 * NW * 16];
    __shared__ int s_wn[NW];
    __shared__ int s_cnt;
    __shared__ uint64_t s_red[2 * NW];
    __shared__ int s_redi[NW];
    __shared__ int s_tie[NQ][NW];
    __shared__ int s_pu, s_yi;
    __shared__ uint64_t s_u;
    const PoolLds L = row_lds(t.S, LS);
    uint64_t* s_top = (uint64_t*)(s_pdyn + L.top);
    uint64_t* s_k2 = (uint64_t*)(s_pdyn + L.k2);
    uint64_t* s_keys = LS ? s_top : s_keys_st;
    int* s_cvi = LS ? (int*)s_k2 : s_cvi_st;

    ieee_mode_off();                             // NaN words drop out of the maxima
    const int tid = threadIdx.x, lane = tid % WAVE, wid = tid / WAVE;
    const int row = blockIdx.x;
    const int b = row / a.P, j = row % a.P;
    const int S = t.S, K = t.K, V = t.V;
    const int level = a.level;
    const int64_t nb = (int64_t)b * t.NN;
    const int NVR = (V + VEC - 1) / VEC;          // vectors of the row, <= NTB * NQ
    const int NVF = V / VEC;                       // whole vectors
    const int nsel = S;                            // S <= V
    const char* base = (const char*)a.logits + (int64_t)row * t.stride * (DT ? 2 : 4);

    // the parent's frontier entry is loaded while the row streams (after
    // its first loads are issued when there are four batches or more), its
    // draw taken while the last batch is in flight, and both checked after
    // the row is streamed
    RowParentRaw rp{0, 0ull};
    bool has_u = false;
    if (tid == 0) s_cnt = 0;
    if (!LS)
        for (int i = tid; i < S; i += NTB) s_top[i] = 0ull;   // id -1 until ranked

    // ---- the row, streamed: vector q of this thread is vidx(q) ------------
    // vm: each vector's maximum -- bf16: the 16-bit order codes of vectors
    // 2 qi (low half) and 2 qi + 1 (high half) in vm[qi]; fp32: its bits
    uint32_t vm[NM];
    uint32_t c1 = 0, c2 = 0, c3 = 0, c4 = 0;
    rs_ushort2 p1 = {0, 0}, p2 = {0, 0};
    // vector q of this thread: lane `lane` of the 64-vector slot (wid + q)
    // mod NW of block stride q.  Rotating the slot spreads every wave's
    // reads over all offsets (mod one block stride, 8 KB) in the row; with
    // a fixed slot per wave its reads kept to one offset, and the waves of
    // a block finished streaming up to several µs apart.
    const int wsu = __builtin_amdgcn_readfirstlane(wid);
    auto vidx = [&](int q) -> int { return (((wsu + q) & (NW - 1)) * WAVE + lane) + NTB * q; };
    auto load_batch = [&](uint4 (&r)[EBATCH], int bt) {
        // plain loads when every lane of the block reads whole vectors
        if (NTB - 1 + NTB * (bt * EBATCH + EBATCH - 1) < NVF) {
#pragma unroll
            for (int e = 0; e < EBATCH; ++e)
                r[e] = load_stream16(base + (int64_t)vidx(bt * EBATCH + e) * 16);
        } else {
#pragma unroll
            for (int e = 0; e < EBATCH; ++e)
                r[e] = load_row_vec<DT>(base, vidx(bt * EBATCH + e), V);
        }
    };
    auto proc_batch = [&](const uint4 (&r)[EBATCH], int bt) {
        if (DT) {
#pragma unroll
            for (int e = 0; e < EBATCH; e += 2) {
                const uint32_t lo = bf16x8_max_raw(r[e]);
                const uint32_t hi = bf16x8_max_raw(r[e + 1]);
                const int qi = (bt * EBATCH + e) / 2;
                const rs_ushort2 cq = bf16x2_codes(__builtin_amdgcn_perm(hi, lo, 0x07060302u));
                vm[qi] = __builtin_bit_cast(uint32_t, cq);
                p2 = __builtin_elementwise_max(p2, __builtin_elementwise_min(p1, cq));
                p1 = __builtin_elementwise_max(p1, cq);
            }
        } else {
#pragma unroll
            for (int e = 0; e < EBATCH; ++e) {
                const float mx = fmaxf(fmaxf(elem<DT>(r[e], 0), elem<DT>(r[e], 1)),
                                       fmaxf(elem<DT>(r[e], 2), elem<DT>(r[e], 3)));
                vm[bt * EBATCH + e] = __float_as_uint(mx);
                const uint32_t cv = ord32(mx) >> 16;
                c4 = max(c4, min(c3, cv));
                c3 = max(c3, min(c2, cv));
                c2 = max(c2, min(c1, cv));
                c1 = max(c1, cv);
            }
        }
    };
    if (NB == 2 && tid == 0) rp = row_parent_load(t, a, b, j);
    {
        uint4 ra[EBATCH], rb[EBATCH];
        load_batch(ra, 0);
#pragma unroll
        for (int bt = 0; bt < NB; bt += 2) {
            load_batch(rb, bt + 1);
            proc_batch(ra, bt);
            if (bt + 2 < NB) load_batch(ra, bt + 2);
            if (NB >= 4 && bt == 0 && tid == 0) rp = row_parent_load(t, a, b, j);
            // the parent's draw (a serial Philox chain) while the last
            // batch is in flight, once the parent's load has returned
            if (bt == NB - 2 && tid == 0 && level > 0) {
                rp.u = parent_draw(a, b, rp.pu);
                has_u = true;
            }
            proc_batch(rb, bt + 1);
        }
    }
    if (tid == 0) row_parent(t, a, b, j, rp, has_u, &s_pu, &s_u);
    // bf16: the two largest of each half (four distinct vectors)
    if (DT) {
        if constexpr (four) {
            c1 = p1.x;
            c2 = p1.y;
            c3 = p2.x;
            c4 = p2.y;
        } else {
            c1 = max((uint32_t)p1.x, (uint32_t)p1.y);
            c2 = max(min((uint32_t)p1.x, (uint32_t)p1.y), max((uint32_t)p2.x, (uint32_t)p2.y));
        }
    }

    // ---- threshold: h = the nsel-th largest of the offered codes (a lower
    //      bound of the nsel-th largest vector maximum)
    uint32_t h = offer_threshold<NTB>(c1, c2, c3, c4, four, nsel, s_thr);
    if constexpr (LS) {
        // raised to the nsel-th largest vector maximum: the high byte of its
        // code, then the low byte, from histograms of the codes >= h
        auto code_of = [&](int q) -> uint32_t {
            if (DT) {
                const rs_ushort2 c = __builtin_bit_cast(rs_ushort2, vm[q / 2]);
                return (q & 1) ? (uint32_t)c.y : (uint32_t)c.x;
            }
            return ord32(__uint_as_float(vm[q])) >> 16;
        };
        for (int i = tid; i < 256; i += NTB) s_hist[i] = 0;
        __syncthreads();
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const uint32_t c = code_of(q);
            if (c >= h && vidx(q) < NVR) atomicAdd(&s_hist[c >> 8], 1);
        }
        __syncthreads();
        const int2 hi8 = suffix_pick256<NTB>(s_hist, nsel, s_thr);
        if (hi8.x >= 0) {
            for (int i = tid; i < 256; i += NTB) s_hist[i] = 0;
            __syncthreads();
#pragma unroll
            for (int q = 0; q < NQ; ++q) {
                const uint32_t c = code_of(q);
                if (c >= h && (int)(c >> 8) == hi8.x && vidx(q) < NVR)
                    atomicAdd(&s_hist[c & 0xFFu], 1);
            }
            __syncthreads();
            const int2 lo8 = suffix_pick256<NTB>(s_hist, nsel - hi8.y, s_thr);
            if (lo8.x >= 0) h = max(h, ((uint32_t)hi8.x << 8) | (uint32_t)lo8.x);
        }
    }
    // the parent record, for the children written at the end
    const ParentRec pr = (tid < K) ? parent_rec(t, level, nb, s_pu) : ParentRec{1.0, 0ull};
    const float tau = (h << 16) > ord32(-INFINITY) ? unord32(h << 16) : -INFINITY;

    // ---- candidate vectors (maximum >= tau): every thread marks its own in
    //      a bit mask (bf16: bit qi is vector 2 qi, bit 16 + qi vector
    //      2 qi + 1; fp32: bit q is vector q), the wave's offsets come from
    //      one prefix sum, and every wave appends them to its region of
    //      s_cvi; if a wave has more than its region holds, but all fit, they
    //      are written again into one list with slots reserved per wave
    constexpr int WCAPR = CV / NW;
    mask_t take = 0;
    {
        // vectors of this thread inside the row: q < nqv
        int nqv = min(NQ, max(0, (NVR - lane - (NTB - WAVE) + NTB - 1) / NTB));
        while (nqv < NQ && vidx(nqv) < NVR) ++nqv;      // at most twice
        if (DT) {
            // code >= h is maximum >= tau, except that a -0 maximum passes
            // tau = +0 as a logit (code of -0: 0x7FFF)
            const uint32_t hc = (h == 0x8000u) ? 0x7FFFu : h;
            const rs_ushort2 h2 = {(unsigned short)hc, (unsigned short)hc};
            const rs_ushort2 one = {1, 1};
            mask_t below = 0;
#pragma unroll
            for (int qi = 0; qi < NM; ++qi) {
                const rs_ushort2 c = __builtin_bit_cast(rs_ushort2, vm[qi]);
                const rs_ushort2 d = __builtin_elementwise_min(__builtin_elementwise_sub_sat(h2, c), one);
                if constexpr (HALF == 16)
                    below |= __builtin_bit_cast(uint32_t, d) << qi;
                else
                    below |= ((mask_t)d.x << qi) | ((mask_t)d.y << (HALF + qi));
            }
            const mask_t vlo = ((mask_t)1 << ((nqv + 1) >> 1)) - 1u;
            const mask_t vhi = (((mask_t)1 << (nqv >> 1)) - 1u) << HALF;
            take = ~below & (vlo | vhi);
        } else {
#pragma unroll
            for (int q = 0; q < NQ; ++q) take |= (mask_t)(__uint_as_float(vm[q]) >= tau) << q;
            take &= nqv >= 8 * (int)sizeof(mask_t) ? ~(mask_t)0 : ((mask_t)1 << nqv) - 1u;
        }
    }
    const int tn = __popcll((uint64_t)take);
    const int texcl = wave_excl_scan(tn);
    auto push_vectors = [&](int pos, int* dst, int cap) {
        for (mask_t mk = take; mk != 0u; mk &= mk - 1u) {
            const int bb = __builtin_ctzll((uint64_t)mk);
            const int q = DT ? ((bb < HALF) ? 2 * bb : 2 * (bb - HALF) + 1) : bb;
            if (pos < cap) dst[pos] = vidx(q);
            ++pos;
        }
    };
    push_vectors(texcl, s_cvi + wid * WCAPR, WCAPR);
    if (lane == WAVE - 1) s_wn[wid] = texcl + tn;
    __syncthreads();
    int wn[NW], nv = 0, wbefore = 0;
    bool ovf = false;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
        wn[w] = s_wn[w];
        ovf |= wn[w] > WCAPR;
        wbefore += (w < wid) ? wn[w] : 0;
        nv += wn[w];
    }
    const bool contig = ovf && nv <= CV;
    if (contig) {
        push_vectors(wbefore + texcl, s_cvi, CV);
        __syncthreads();
    }
    // ---- their elements >= tau (candidate vectors read again, one per
    //      thread and round; small supports have a single round)
    auto gather = [&](int e) {
        uint4 x = make_uint4(0, 0, 0, 0);
        int e0 = V;
        if (e < nv) {
            // entry e of the concatenated regions (or of the one list)
            int w = 0, off = e;
            if (!contig) {
#pragma unroll
                for (int q = 0; q < NW - 1; ++q) {
                    const bool past = off >= wn[q] && w == q;
                    off -= past ? wn[q] : 0;
                    w += past ? 1 : 0;
                }
            }
            const int vi = s_cvi[w * WCAPR + off];
            x = load_row_vec<DT>(base, vi, V);
            e0 = vi * VEC;
        }
        int n = 0;
#pragma unroll
        for (int k = 0; k < VEC; ++k) n += (elem<DT>(x, k) >= tau) & (e0 + k < V);
        const int excl = wave_excl_scan(n);
        int cb = 0;
        if (lane == WAVE - 1) cb = atomicAdd(&s_cnt, excl + n);
        int pos = (int)lane_u32((uint32_t)cb, WAVE - 1) + excl;
#pragma unroll
        for (int k = 0; k < VEC; ++k) {
            const float v = elem<DT>(x, k);
            if (v >= tau && e0 + k < V) {
                if (pos < CC) s_keys[pos] = logit_key(v, (uint32_t)(e0 + k));
                ++pos;
            }
        }
    };
    if (!ovf || contig) {
        if constexpr (LS || CAPV > NTB) {
            for (int e = tid; e - tid < nv; e += NTB) gather(e);
        } else {
            gather(tid);                          // nv <= CAPV <= NTB
        }
    } else if (tid == 0) {
        s_cnt = CC + 1;                          // too many: exact fallback below
    }
    __syncthreads();
    int cnt = s_cnt;
    if (cnt > CC) {
        __syncthreads();
        if (tid == 0) s_cnt = 0;
        exact_select_fallback<DT, NTB, NQ>(
            base, V, 0, h, nsel, CC,
            [=](float v, int id) {
                const int pos = atomicAdd(&s_cnt, 1);
                if (pos < CC) s_keys[pos] = logit_key(v, (uint32_t)id);
            },
            s_redi, s_tie);
        cnt = min(fallback_count(&s_cnt), CC);
    }

    // ---- the support: the top nsel candidates in (logit desc, id asc) order
    if constexpr (LS) {
        // sorted in place (padding 0 sorts last; at least nsel entries)
        const int n2 = pow2_at_least(max(cnt, nsel));
        for (int i = cnt + tid; i < n2; i += NTB) s_keys[i] = 0ull;
        __syncthreads();
        bitonic_sort_desc<NTB>(s_keys, n2);
    } else {
        rank_keys<NTB>(s_keys, cnt, s_rank, s_top, nsel);     // placed as ranked
    }
    __syncthreads();

    pool_form<NTB>(t, a, row, s_pdyn, L, s_pu, pr, s_u, s_red, &s_yi);
    if (level + 1 >= t.D) return;
    select_frontier(t, a, b, s_top, s_k2);
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
    const size_t shm = (size_t)pool_lds(t.S, t.C).bytes;
    k_pool<<<t.B * a.P, NTP, shm, s>>>(t, a);
    return hipGetLastError();
}

int expand_variant_nvc(int v) { return kNVC[v]; }

// ---------------------------------------------------------------------------
// k_row_wsum: for the whole-vocabulary construction of a sparse tree, the
// total construction weight of every row of the level, sum over all V of
// w(l; M, k1) with M the row maximum (the same weights the pool computes
// on its support).  One block per row, two passes over the row: the
// maximum, then the weights.
// ---------------------------------------------------------------------------
constexpr int NTW = 256;

template <int DT>
__global__ __launch_bounds__(NTW) void k_row_wsum(TreeDev t, LevelArgs a) {
    constexpr int VEC = DT ? 8 : 4;
    __shared__ float s_max[NTW / WAVE];
    __shared__ uint64_t s_sum[NTW / WAVE];
    const int row = blockIdx.x;
    const int V = t.V;
    const int NVR = (V + VEC - 1) / VEC;
    const char* base = (const char*)a.logits + (int64_t)row * t.stride * (DT ? 2 : 4);
    float mx = -INFINITY;
    for (int vi = threadIdx.x; vi < NVR; vi += NTW) {
        const uint4 x = load_row_vec<DT>(base, vi, V);
#pragma unroll
        for (int k = 0; k < VEC; ++k)
            if (vi * VEC + k < V) mx = fmaxf(mx, elem<DT>(x, k));
    }
    const float M = block_max<NTW>(mx, s_max);
    uint64_t sum = 0;
    for (int vi = threadIdx.x; vi < NVR; vi += NTW) {
        const uint4 x = load_row_vec<DT>(base, vi, V);
#pragma unroll
        for (int k = 0; k < VEC; ++k)
            if (vi * VEC + k < V) sum += cweight(elem<DT>(x, k), M, a.k1);
    }
    sum = block_sum_u64<NTW>(sum, s_sum);
    if (threadIdx.x == 0) t.s1row[row] = sum;
}

hipError_t launch_row_wsum(const TreeDev& t, const LevelArgs& a, hipStream_t s) {
    const dim3 grid(t.B * a.P);
    if (t.dtype) k_row_wsum<1><<<grid, NTW, 0, s>>>(t, a);
    else k_row_wsum<0><<<grid, NTW, 0, s>>>(t, a);
    return hipGetLastError();
}

// Vectors per thread k_expand_row needs for a row of V elements (16, 32 or 48),
// or 0 if the row is too long for it.
int expand_row_nq(int dtype, int V) {
    const int nvr = (V + (dtype ? 8 : 4) - 1) / (dtype ? 8 : 4);
    if (nvr <= NTE * 16) return 16;
    if (nvr <= NTE * 32) return 32;
    if (nvr <= NTE * 48) return 48;
    return 0;
}

// A level of more rows than the device holds 512-thread blocks at once
// runs 256-thread blocks with twice the vectors per thread (rows of up to
// 32 vectors per 512 threads), which the device holds twice as many of: the
// rows past the first round no longer wait for a whole block to end.
static bool row_narrow(const TreeDev& t, int rows, int nq) {
    if (nq > 32) return false;
    if (t.row_narrow >= 0) return t.row_narrow == 1;
    return t.row_slots > 0 && rows > t.row_slots;
}

template <int DT, int SC>
static hipError_t launch_row(const TreeDev& t, const LevelArgs& a, int nq, hipStream_t s) {
    const dim3 grid(t.B * a.P);
    const size_t shm = (size_t)row_lds(t.S, SC == 2).bytes;
    const bool narrow = row_narrow(t, t.B * a.P, nq);
    if (narrow && nq == 32)
        k_expand_row<DT, 64, SC, NTE / 2><<<grid, NTE / 2, shm, s>>>(t, a);
    else if (narrow && nq == 16)
        k_expand_row<DT, 32, SC, NTE / 2><<<grid, NTE / 2, shm, s>>>(t, a);
    else if (nq == 16) k_expand_row<DT, 16, SC, NTE><<<grid, NTE, shm, s>>>(t, a);
    else if (nq == 32) k_expand_row<DT, 32, SC, NTE><<<grid, NTE, shm, s>>>(t, a);
    else if (nq == 48) k_expand_row<DT, 48, SC, NTE><<<grid, NTE, shm, s>>>(t, a);
    else return hipErrorInvalidValue;
    return hipGetLastError();
}

template <int DT>
static hipError_t launch_row_dt(const TreeDev& t, const LevelArgs& a, int nq, hipStream_t s) {
    if (t.S > kLargeSupport) return launch_row<DT, 2>(t, a, nq, s);
    if (t.S > NTE / 4) return launch_row<DT, 1>(t, a, nq, s);
    return launch_row<DT, 0>(t, a, nq, s);
}

template <int DT, int SC>
static const void* row_fn(int nq) {
    if (nq == 16) return (const void*)&k_expand_row<DT, 16, SC, NTE>;
    if (nq == 32) return (const void*)&k_expand_row<DT, 32, SC, NTE>;
    if (nq == 48) return (const void*)&k_expand_row<DT, 48, SC, NTE>;
    return nullptr;
}

template <int DT>
static const void* row_fn_dt(int S, int nq) {
    if (S > kLargeSupport) return row_fn<DT, 2>(nq);
    if (S > NTE / 4) return row_fn<DT, 1>(nq);
    return row_fn<DT, 0>(nq);
}

// How many 512-thread blocks of this tree's row kernel the device holds at
// once (0 when the rows are too long for the row kernel).
hipError_t expand_row_slots(const TreeDev& t, int* slots) {
    *slots = 0;
    const int nq = expand_row_nq(t.dtype, t.V);
    const void* fn = t.dtype ? row_fn_dt<1>(t.S, nq) : row_fn_dt<0>(t.S, nq);
    if (!fn) return hipSuccess;
    int dev = 0, cus = 0, per = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e == hipSuccess)
        e = hipOccupancyMaxActiveBlocksPerMultiprocessor(
            &per, fn, NTE, (size_t)row_lds(t.S, t.S > kLargeSupport).bytes);
    if (e == hipSuccess) *slots = per * cus;
    return e;
}

hipError_t launch_expand_row(const TreeDev& t, const LevelArgs& a, hipStream_t s) {
    const int nq = expand_row_nq(t.dtype, t.V);
    return t.dtype ? launch_row_dt<1>(t, a, nq, s) : launch_row_dt<0>(t, a, nq, s);
}

}  // namespace rheo
