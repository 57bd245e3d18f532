// RheoVerification (Algorithm 1) applied layer by layer from the root of the
// pruned tree (Thm. 1).  One block walks one sequence.
//
// Per layer, at the current node u:
//   p = softmax(target(u) / T) over the whole vocabulary, as canonical
//   integer weights P_v (relative to the row maximum) with the exact total
//   S_p and the totals of fixed 64*VEC-token chunks (for the inverse CDF).
//   Candidates C = children of u in the pruned tree, in slot order; s = the
//   sampled child's position or -1.
//   s != -1: accept Y iff eta <= p(Y) / q~(Y), i.e.
//            (U+1) Q_Y S_p <= 2^32 P_Y Z_q;  else drop Y and take the residual
//            r_v ~ N_v = max(0, P_v Z_q - Q_v S_p)  (q~ is the truncated tail
//            stored at expansion; N_v = P_v Z_q off its support).
//   s == -1: r_v ~ N_v = P_v.
//   Each remaining candidate in slot order is accepted iff
//   (U+1) Z_rem <= 2^32 N_u, else N_u = 0 and Z_rem -= N_u.
//   If none is accepted (or C is empty), u* ~ r by inverse CDF over token ids:
//   t = floor(U64 Z_rem / 2^64), the chunk holding t from the chunk totals
//   corrected at the overridden tokens, then a scan of that chunk.
// All tests are exact integer comparisons (eta = (U+1) / 2^32 in (0, 1]).
#include "rheo_device.h"
#include "rheo_state.h"

namespace rheo {

constexpr int NCMAX = 1024;      // chunks: V <= 262143, chunk >= 256 tokens
constexpr int SPMAX = 1024 + 16; // overridden tokens: support tail + candidates

template <int DT>
__device__ __forceinline__ float load_logit(const char* row, int v) {
    if (DT) return __uint_as_float((uint32_t)((const uint16_t*)row)[v] << 16);
    return ((const float*)row)[v];
}

template <int DT>
__device__ __forceinline__ float velem(const uint4& v, int k) {
    const uint32_t* w = &v.x;
    if (DT) return (k & 1) ? bf_hi(w[k >> 1]) : bf_lo(w[k >> 1]);
    return __uint_as_float(w[k]);
}

template <int DT>
__device__ __forceinline__ uint4 load_vec(const char* row, int vi, int V) {
    constexpr int VEC = DT ? 8 : 4;
    constexpr int ESZ = DT ? 2 : 4;
    const int e = vi * VEC;
    if (e + VEC <= V) return *(const uint4*)(row + (int64_t)e * ESZ);
    uint32_t w[4];
    if (DT) {
        const uint16_t* p = (const uint16_t*)row;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const uint32_t lo = (e + 2 * q < V) ? p[e + 2 * q] : 0xFF80u;
            const uint32_t hi = (e + 2 * q + 1 < V) ? p[e + 2 * q + 1] : 0xFF80u;
            w[q] = lo | (hi << 16);
        }
    } else {
        const uint32_t* p = (const uint32_t*)row;
#pragma unroll
        for (int q = 0; q < 4; ++q) w[q] = (e + q < V) ? p[e + q] : 0xFF800000u;
    }
    return make_uint4(w[0], w[1], w[2], w[3]);
}

// Position of token v in the id-sorted tail list, -1 if absent.
__device__ inline int find_sorted(const int32_t* ids, int n, int v) {
    int lo = 0, hi = n;
    while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (ids[mid] < v) lo = mid + 1; else hi = mid;
    }
    return (lo < n && ids[lo] == v) ? lo : -1;
}

template <int DT, int NT>
__global__ __launch_bounds__(NT) void k_verify(TreeDev t, VerifyArgs a) {
    constexpr int VEC = DT ? 8 : 4;
    constexpr int CH = WAVE * VEC;

    __shared__ uint64_t s_chunk[NCMAX];
    __shared__ u128 s_def[NCMAX];
    __shared__ int32_t s_sp_id[SPMAX];
    __shared__ uint32_t s_sp_P[SPMAX];
    __shared__ u128 s_sp_N[SPMAX];
    __shared__ u128 s_cn[CH];
    __shared__ int16_t s_mark[CH];
    __shared__ int s_c_uid[16], s_c_tok[16], s_c_slot[16], s_c_kind[16];
    __shared__ uint32_t s_c_P[16];
    __shared__ float s_redf[NT / WAVE];
    __shared__ uint64_t s_red[NT / WAVE];
    __shared__ int s_nc, s_spos, s_e, s_nsp, s_done, s_next, s_token, s_cstar;
    __shared__ u128 s_F, s_tt;

    const int tid = threadIdx.x;
    const int lane = tid % WAVE, wid = tid / WAVE;
    const int b = blockIdx.x;
    const int V = t.V, K = t.K, NN = t.NN;
    const int nvec = (V + VEC - 1) / VEC;
    const int NC = (V + CH - 1) / CH;
    const int64_t nb = (int64_t)b * NN;
    const int nt = t.S - t.m;             // entries of a stored tail list

    int cur = 0;                          // uid of the current node
    int level = 0;
    int nacc = 0;
    for (;;) {
        if (level > t.D) {                 // unreachable: every accept descends
            if (tid == 0) atomicOr(t.err, 32);
            break;
        }
        int cur_p = t.pidx[nb + cur];
        if (cur_p < 0 || cur_p > a.R) {
            if (tid == 0) atomicOr(t.err, 32);
            cur_p = 0;
        }
        const char* row = (const char*)a.logits +
                          ((int64_t)b * (a.R + 1) + cur_p) * t.stride * (DT ? 2 : 4);
        // ---- candidates of this layer ----------------------------------
        if (tid == 0) {
            int nc = 0, spos = -1;
            const int fc = t.first_child[nb + cur];
            if (fc >= 0) {
                for (int sl = 0; sl < K; ++sl) {
                    const int c = fc + sl;
                    if (t.pidx[nb + c] > 0) {
                        const int kind = (t.meta[nb + c] >> 16) & 0xFF;
                        if (kind == SAMPLED) spos = nc;
                        s_c_uid[nc] = c;
                        s_c_tok[nc] = t.tok[nb + c];
                        s_c_slot[nc] = sl + 1;
                        s_c_kind[nc] = kind;
                        ++nc;
                    }
                }
            }
            s_nc = nc;
            s_spos = spos;
            s_e = t.exp_of[nb + cur];
        }
        // ---- pass A: row maximum ----------------------------------------
        float mx = -INFINITY;
        for (int vi = tid; vi < nvec; vi += NT) {
            const uint4 x = load_vec<DT>(row, vi, V);
#pragma unroll
            for (int k = 0; k < VEC; ++k) mx = fmaxf(mx, velem<DT>(x, k));
        }
        const float M = block_max<NT>(mx, s_redf);
        // ---- pass B: weights, chunk totals --------------------------------
        const int iters = (nvec + NT - 1) / NT;
        for (int it = 0; it < iters; ++it) {
            const int vi = it * NT + tid;
            uint64_t sum = 0;
            if (vi < nvec) {
                const uint4 x = load_vec<DT>(row, vi, V);
#pragma unroll
                for (int k = 0; k < VEC; ++k) {
                    const int v = vi * VEC + k;
                    if (v < V) sum += cweight(velem<DT>(x, k), M, a.kT);
                }
            }
            sum = wave_sum_u64(sum);
            const int c = it * (NT / WAVE) + wid;
            if (lane == 0 && c < NC) s_chunk[c] = sum;
        }
        __syncthreads();
        uint64_t part = 0;
        for (int c = tid; c < NC; c += NT) part += s_chunk[c];
        const uint64_t Sp = block_sum_u64<NT>(part, s_red);
        // ---- gathers: P at the candidates and on the stored tail ---------
        const int nc = s_nc, spos = s_spos, e = s_e;
        if (tid < nc) s_c_P[tid] = cweight(load_logit<DT>(row, s_c_tok[tid]), M, a.kT);
        if (spos >= 0) {
            const int64_t tb = ((int64_t)b * t.E + e) * t.S;
            for (int i = tid; i < nt; i += NT) {
                const int v = t.tail_id[tb + i];
                s_sp_id[i] = v;
                s_sp_P[i] = cweight(load_logit<DT>(row, v), M, a.kT);
            }
        }
        __syncthreads();
        // ---- Algorithm 1 at this layer (one thread, exact integers) -------
        if (tid == 0) {
            int done = 0, next = -1, token = -1, nsp = 0;
            u128 F = 1, Zrem = Sp;
            bool sampled_rejected = false;
            if (spos >= 0) {
                const int64_t tb = ((int64_t)b * t.E + e) * t.S;
                const uint64_t Zq = t.zq[(int64_t)b * t.E + e];
                const int yi = find_sorted(s_sp_id, nt, s_c_tok[spos]);
                const uint64_t QY = (yi >= 0) ? t.tail_q[tb + yi] : 0;
                const uint64_t PY = s_c_P[spos];
                const uint64_t U = philox_draw(a.rng_key, P_VERIFY, (uint64_t)b,
                                               (uint64_t)(32 * level)) >> 32;
                const u128 lhs = (u128)(U + 1) * QY * Sp;
                const u128 rhs = ((u128)PY * Zq) << 32;
                if (yi < 0) atomicOr(t.err, 4);
                if (lhs <= rhs) {
                    next = s_c_uid[spos];
                    token = s_c_tok[spos];
                } else {
                    sampled_rejected = true;
                    F = Zq;
                    u128 def = 0;
                    for (int i = 0; i < nt; ++i) {
                        const u128 pz = (u128)s_sp_P[i] * Zq;
                        const u128 qs = (u128)t.tail_q[tb + i] * Sp;
                        const u128 nv = pz > qs ? pz - qs : (u128)0;
                        s_sp_N[i] = nv;
                        def += pz - nv;
                    }
                    nsp = nt;
                    Zrem = (u128)Zq * Sp - def;
                }
            }
            if (next < 0) {
                for (int ci = 0; ci < nc; ++ci) {
                    if (ci == spos) continue;
                    const int tok = s_c_tok[ci];
                    int sp = sampled_rejected ? find_sorted(s_sp_id, nt, tok) : -1;
                    const u128 Nu = (sp >= 0) ? s_sp_N[sp] : F * (u128)s_c_P[ci];
                    const uint64_t U = philox_draw(a.rng_key, P_VERIFY, (uint64_t)b,
                                                   (uint64_t)(32 * level + s_c_slot[ci])) >> 32;
                    if ((u128)(U + 1) * Zrem <= (Nu << 32)) {
                        next = s_c_uid[ci];
                        token = tok;
                        break;
                    }
                    Zrem -= Nu;
                    if (sp >= 0) {
                        s_sp_N[sp] = 0;
                    } else {
                        s_sp_id[nsp] = tok;
                        s_sp_P[nsp] = s_c_P[ci];
                        s_sp_N[nsp] = 0;
                        ++nsp;
                    }
                }
            }
            if (next < 0) {
                done = 1;
                const uint64_t U = philox_draw(a.rng_key, P_FINAL, (uint64_t)b, (uint64_t)level);
                s_tt = mulhi_64x128(U, Zrem);
            }
            s_done = done;
            s_next = next;
            s_token = token;
            s_nsp = nsp;
            s_F = F;
        }
        __syncthreads();
        if (!s_done) {
            if (tid == 0) a.accepted[(int64_t)b * t.D + nacc] = s_token;
            ++nacc;
            cur = s_next;
            ++level;
            __syncthreads();
            continue;
        }
        // ---- final sample u* ~ r by inverse CDF over token ids -------------
        const int nsp = s_nsp;
        const u128 F = s_F;
        for (int c = tid; c < NC; c += NT) s_def[c] = 0;
        __syncthreads();
        if (tid == 0) {
            for (int i = 0; i < nsp; ++i)
                s_def[s_sp_id[i] / CH] += F * (u128)s_sp_P[i] - s_sp_N[i];
            u128 acc = 0;
            const u128 tt = s_tt;
            int cs = NC - 1;
            for (int c = 0; c < NC; ++c) {
                const u128 w = F * (u128)s_chunk[c] - s_def[c];
                if (acc + w > tt) { cs = c; break; }
                acc += w;
            }
            s_cstar = cs;
            s_tt = tt - acc;
        }
        for (int i = tid; i < CH; i += NT) s_mark[i] = -1;
        __syncthreads();
        const int cs = s_cstar;
        for (int i = tid; i < nsp; i += NT)
            if (s_sp_id[i] / CH == cs) s_mark[s_sp_id[i] - cs * CH] = (int16_t)i;
        __syncthreads();
        for (int i = tid; i < CH; i += NT) {
            const int v = cs * CH + i;
            u128 w = 0;
            if (v < V) {
                const int mk = s_mark[i];
                w = (mk >= 0) ? s_sp_N[mk] : F * (u128)cweight(load_logit<DT>(row, v), M, a.kT);
            }
            s_cn[i] = w;
        }
        __syncthreads();
        if (tid == 0) {
            u128 acc = 0;
            const u128 tt = s_tt;
            int tok = -1;
            for (int i = 0; i < CH; ++i) {
                acc += s_cn[i];
                if (acc > tt) { tok = cs * CH + i; break; }
            }
            if (tok < 0) atomicOr(t.err, 8);
            a.final_token[b] = tok;
            a.accept_len[b] = nacc;
            for (int i = nacc; i < t.D; ++i) a.accepted[(int64_t)b * t.D + i] = -1;
        }
        break;
    }
}

hipError_t launch_verify(const TreeDev& t, const VerifyArgs& a, hipStream_t s) {
    if (t.dtype) k_verify<1, 1024><<<t.B, 1024, 0, s>>>(t, a);
    else k_verify<0, 1024><<<t.B, 1024, 0, s>>>(t, a);
    return hipGetLastError();
}

}  // namespace rheo
