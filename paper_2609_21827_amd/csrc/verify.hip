// RheoVerification (Algorithm 1) applied layer by layer from the root of the
// pruned tree (Thm. 1).
//
// A team of G co-resident blocks walks one sequence (the grid never exceeds
// what the device holds at once; see launch_verify).
// At each layer the current node's target row is split into G segments of
// whole 64*VEC-token chunks; every block holds its segment in registers:
//   1. the row maximum M: every block reads the target logits at all
//      special tokens (the children, and in sparse mode the stored tail of
//      q~) and takes their maximum as a guess of M, which step 2 uses and
//      checks: M is at least the guess, and equals it when no segment
//      exceeds it (nearly always: the target's argmax is almost always
//      among the draft's top tokens); otherwise M is exchanged and step 2
//      repeated
//   2. canonical weights P_v of p = softmax(target / T) (relative to M) for
//      the segment, the totals of its chunks, and P at the special tokens
//      -> team exchange of the segment sums, with the guess's check
//   3. every block takes the same Algorithm 1 decision from the exchanged
//      totals with exact integer tests:
//        s != -1: accept Y iff (U+1) Q_Y S_p <= 2^32 P_Y Z_q; otherwise the
//                 residual r ~ N_v = max(0, P_v Z_q - Q_v S_p) (Q_v = 0 off
//                 the stored tail), with total
//                 Z_r = Z_q S_p - sum_tail min(P_v Z_q, Q_v S_p);
//        s == -1: r ~ N_v = P_v;
//        each remaining candidate in slot order: accept iff
//        (U+1) Z_rem <= 2^32 N_u, else N_u = 0, Z_rem -= N_u;
//        none accepted (or no candidates): u* ~ r by inverse CDF over token
//        ids, t = floor(U64 Z_rem / 2^64): the chunk holding t from the chunk
//        totals corrected at the special tokens, then a scan of that chunk.
//      The RRSw baseline (App. D.2) tests the leads -- the candidates before
//      the sampled child -- first, under p; then the sampled child against
//      what remains (mass Z_l = S_p less the rejected leads) in place of S_p
//      above, and the fills under the residual with Z_l for S_p.
// Team exchanges use agent-scope atomic stores and loads only (they are
// coherent across the XCDs without cache write-back or invalidation), with
// arrival epochs in per-block flags and bounded waits.  The epochs of a
// launch come from a per-team ticket counter in device memory: each block
// of the team takes one ticket as it starts, so the G blocks of the n-th
// launch for that team hold tickets nG .. nG + G - 1 and all compute n,
// whatever order they start in, and the next launch on the stream (which
// starts only after every block of this one has ended) computes n + 1.
// Replays of a captured graph therefore never see their own earlier
// words as current, and no block depends on another block's progress to
// learn the epoch.  A wait past its spin limit ends
// the walk: the team's first block then writes the failure result
// (accept_len = final_token = -1, accepted all -1) and device error bit 128
// is set.  A visited node whose target row has no finite logit (p
// undefined) ends the walk with the same result and device error bit 512.
#include <cstdlib>

#include "rheo_device.h"
#include "rheo_state.h"

namespace rheo {

constexpr int NTV = 256;
constexpr int NWV = NTV / WAVE;
constexpr int GMAX = 64;
constexpr int NCMAX = 1024;      // chunks: V <= 262143, chunk >= 256 tokens
constexpr int SPMAX = 1024 + 16; // stored tail + candidates

template <int DT>
__device__ __forceinline__ float velem(const uint4& v, int k) {
    const uint32_t* w = &v.x;
    if (DT) return (k & 1) ? bf_hi(w[k >> 1]) : bf_lo(w[k >> 1]);
    return __uint_as_float(w[k]);
}

template <int DT>
__device__ __forceinline__ float load_logit(const char* row, int v) {
    if (DT) return __uint_as_float((uint32_t)((const uint16_t*)row)[v] << 16);
    return ((const float*)row)[v];
}

template <int DT>
__device__ __forceinline__ uint4 load_vec(const char* row, int vi, int V) {
    constexpr int VEC = DT ? 8 : 4;
    constexpr int ESZ = DT ? 2 : 4;
    const int e = vi * VEC;
    if (e + VEC <= V) return load_stream16(row + (int64_t)e * ESZ);
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

// 128-bit wave / block sums and scans (values < 2^127), on DPP row moves
// with explicit carries between the 64-bit halves.
__device__ __forceinline__ void add_u128(uint64_t& lo, uint64_t& hi, uint64_t blo, uint64_t bhi) {
    const uint64_t n = lo + blo;
    hi += bhi + (n < lo ? 1ull : 0ull);
    lo = n;
}
__device__ __forceinline__ u128 wave_sum_u128(u128 v) {
    uint64_t lo = (uint64_t)v, hi = (uint64_t)(v >> 64);
    add_u128(lo, hi, row_ror64<8>(lo), row_ror64<8>(hi));
    add_u128(lo, hi, row_ror64<4>(lo), row_ror64<4>(hi));
    add_u128(lo, hi, row_ror64<2>(lo), row_ror64<2>(hi));
    add_u128(lo, hi, row_ror64<1>(lo), row_ror64<1>(hi));
    uint64_t rlo = lane_u64(lo, 0), rhi = lane_u64(hi, 0);
    add_u128(rlo, rhi, lane_u64(lo, 16), lane_u64(hi, 16));
    add_u128(rlo, rhi, lane_u64(lo, 32), lane_u64(hi, 32));
    add_u128(rlo, rhi, lane_u64(lo, 48), lane_u64(hi, 48));
    return ((u128)rhi << 64) | rlo;
}
__device__ __forceinline__ u128 wave_incl_scan_u128(u128 v) {
    const int row = (threadIdx.x % WAVE) >> 4;
    uint64_t lo = (uint64_t)v, hi = (uint64_t)(v >> 64);
    add_u128(lo, hi, row_shr64<1>(lo), row_shr64<1>(hi));
    add_u128(lo, hi, row_shr64<2>(lo), row_shr64<2>(hi));
    add_u128(lo, hi, row_shr64<4>(lo), row_shr64<4>(hi));
    add_u128(lo, hi, row_shr64<8>(lo), row_shr64<8>(hi));
    const uint64_t l0 = lane_u64(lo, 15), h0 = lane_u64(hi, 15);
    const uint64_t l1 = lane_u64(lo, 31), h1 = lane_u64(hi, 31);
    const uint64_t l2 = lane_u64(lo, 47), h2 = lane_u64(hi, 47);
    if (row >= 1) add_u128(lo, hi, l0, h0);
    if (row >= 2) add_u128(lo, hi, l1, h1);
    if (row >= 3) add_u128(lo, hi, l2, h2);
    return ((u128)hi << 64) | lo;
}
// exclusive scan across the block; *total receives the sum
__device__ u128 block_excl_scan_u128(u128 v, u128* sh, u128* total) {
    const int l = threadIdx.x % WAVE, w = threadIdx.x / WAVE;
    const u128 inc = wave_incl_scan_u128(v);
    __syncthreads();
    if (l == WAVE - 1) sh[w] = inc;
    __syncthreads();
    u128 base = 0, tot = 0;
#pragma unroll
    for (int i = 0; i < NWV; ++i) {
        if (i < w) base += sh[i];
        tot += sh[i];
    }
    *total = tot;
    return base + inc - v;
}
__device__ u128 block_sum_u128(u128 v, u128* sh) {
    const int l = threadIdx.x % WAVE, w = threadIdx.x / WAVE;
    v = wave_sum_u128(v);
    __syncthreads();
    if (l == 0) sh[w] = v;
    __syncthreads();
    u128 tot = 0;
#pragma unroll
    for (int i = 0; i < NWV; ++i) tot += sh[i];
    return tot;
}

// Team barrier: publish this block's arrival at `epoch`, then wait until
// every team member has arrived.  Prior team-visible stores must be agent
// atomic stores; each thread waits for its own before the block barrier.
// Returns false (and raises the error flag) if the wait timed out.
// The team's row maximum: every block publishes its segment maximum in one
// word with the (low 32 bits of the) epoch, and waits until all G words of
// the team carry that epoch; the words then hold every segment's maximum,
// so no separate barrier or read follows.  *s_M receives the maximum.
// Bounded like team_barrier.
__device__ bool team_max_exchange(uint64_t* words, int g, int G, uint64_t epoch, float mx,
                                  long spin_limit, int32_t* err, int* s_ok, float* s_M) {
    const uint32_t e32 = (uint32_t)epoch;
    if (threadIdx.x < WAVE) {
        if (threadIdx.x == 0) {
            *s_ok = 1;
            __hip_atomic_store(&words[g], ((uint64_t)e32 << 32) | ord32(mx), __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
        }
        float v = -INFINITY;
        long spins = 0;
        for (;;) {
            bool ok = true;
            if ((int)threadIdx.x < G) {
                const uint64_t w = __hip_atomic_load(&words[threadIdx.x], __ATOMIC_RELAXED,
                                                     __HIP_MEMORY_SCOPE_AGENT);
                ok = (uint32_t)(w >> 32) == e32;
                v = unord32((uint32_t)w);
            }
            if (__all(ok)) break;
            if (++spins > spin_limit) {
                if (threadIdx.x == 0) {
                    atomicOr(err, 128);
                    *s_ok = 0;
                }
                break;
            }
            __builtin_amdgcn_s_sleep(1);
        }
        v = wave_max(v);
        if (threadIdx.x == 0) *s_M = v;
    }
    __syncthreads();
    return *s_ok != 0;
}

// The team's total of p's weights (sparse mode): every block publishes the
// sum over its segment (< 2^48 - 1: at most 2^18 - 1 tokens of weight
// <= 2^30) in one word with the low 16 bits of the epoch, after its chunk
// totals; the words then carry every segment's sum, so the total needs no
// further read.  A block whose weights were taken relative to a guessed
// maximum that its segment exceeds publishes 2^48 - 1 instead (no sum
// reaches it), and *s_miss tells every block of the team.  A word left from
// an earlier barrier is fewer than 2^16 epochs old, so the 16-bit
// comparison cannot mistake it for the current one.  wsum holds the block's
// per-wave sums, kMiss for a wave that saw the guess exceeded.  Bounded like
// team_barrier.
constexpr uint64_t kMiss = (1ull << 48) - 1;

__device__ bool team_sum_exchange(uint64_t* words, int g, int G, uint64_t epoch,
                                  const uint64_t* wsum, int nw, long spin_limit, int32_t* err,
                                  int* s_ok, uint64_t* s_total, int* s_miss) {
    constexpr uint64_t M48 = (1ull << 48) - 1;
    const uint64_t e16 = epoch & 0xFFFFull;
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x < WAVE) {
        if (threadIdx.x == 0) {
            *s_ok = 1;
            uint64_t sum = 0;
            bool miss = false;
            for (int w = 0; w < nw; ++w) {
                miss |= wsum[w] == kMiss;
                sum += wsum[w];
            }
            __hip_atomic_store(&words[g], (e16 << 48) | (miss ? kMiss : sum & M48),
                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        uint64_t v = 0;
        bool miss = false;
        long spins = 0;
        for (;;) {
            bool ok = true;
            if ((int)threadIdx.x < G) {
                const uint64_t w = __hip_atomic_load(&words[threadIdx.x], __ATOMIC_RELAXED,
                                                     __HIP_MEMORY_SCOPE_AGENT);
                ok = (w >> 48) == e16;
                v = w & M48;
                miss = v == kMiss;
            }
            if (__all(ok)) break;
            if (++spins > spin_limit) {
                if (threadIdx.x == 0) {
                    atomicOr(err, 128);
                    *s_ok = 0;
                }
                break;
            }
            __builtin_amdgcn_s_sleep(1);
        }
        const bool any_miss = __ballot(miss) != 0;
        v = wave_sum_u64(v);
        if (threadIdx.x == 0) {
            *s_total = v;
            *s_miss = any_miss ? 1 : 0;
        }
    }
    __syncthreads();
    return *s_ok != 0;
}

__device__ bool team_barrier(uint64_t* flags, int g, int G, uint64_t epoch, long spin_limit,
                             int32_t* err, int* s_ok) {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x < WAVE) {
        if (threadIdx.x == 0) {
            *s_ok = 1;
            __hip_atomic_store(&flags[g], epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        long spins = 0;
        for (;;) {
            bool ok = true;
            if ((int)threadIdx.x < G)
                ok = __hip_atomic_load(&flags[threadIdx.x], __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT) >= epoch;
            if (__all(ok)) break;
            if (++spins > spin_limit) {
                if (threadIdx.x == 0) {
                    atomicOr(err, 128);
                    *s_ok = 0;
                }
                break;
            }
            __builtin_amdgcn_s_sleep(1);
        }
    }
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __syncthreads();
    return *s_ok != 0;
}

// At least four blocks per compute unit (128 registers a lane): the team
// shape is sized from how many blocks the device holds at once.
template <int DT, int DN>
__global__ __launch_bounds__(NTV, 4) void k_verify(TreeDev t, VerifyArgs a) {
    constexpr int VEC = DT ? 8 : 4;
    constexpr int ESZ = DT ? 2 : 4;
    constexpr int CH = WAVE * VEC;           // tokens per chunk
    constexpr int JREG = 4;                  // chunks per wave held in registers
    const int SEGCH = a.NV;                  // chunks per segment

    __shared__ uint64_t s_chunk[NCMAX];
    __shared__ __align__(16) int32_t s_tid[SPMAX];   // stored tail ids (rank order)
    __shared__ uint32_t s_tq[SPMAX];         // stored tail weights Q
    __shared__ uint32_t s_tp[SPMAX];         // p's weights at tail tokens, then candidates
    // the chunk scan of the final sample (s_cn), and before it the live
    // tail tokens' deficits of every chunk in two limbs (s_dlo, s_dhi)
    __shared__ __align__(16) uint64_t s_scr[2 * NCMAX];
    static_assert(2 * CH <= 2 * NCMAX, "s_cn fits the scratch");
    u128* const s_cn = (u128*)s_scr;
    uint64_t* const s_dlo = s_scr;
    uint64_t* const s_dhi = s_scr + NCMAX;
    __shared__ u128 s_w128[NWV];
    __shared__ uint64_t s_red[NWV];
    __shared__ float s_redf[NWV];
    __shared__ int s_c_uid[16], s_c_tok[16], s_c_slot[16], s_c_tail[16], s_c_zero[16];
    __shared__ int s_c_pidx[16], s_c_fc[16], s_c_e[16];   // candidates' pruned index, first
                                                           // child and expanded index
    __shared__ uint32_t s_c_q[16];               // dense: q~ weights of the candidates
    __shared__ int s_lead[16];                   // dense: the node's leads
    __shared__ int s_nc, s_spos, s_mode, s_next, s_token, s_cstar;
    __shared__ int s_cur, s_curp, s_fc, s_e;     // the node this layer verifies
    __shared__ int s_resid;                      // the sampled child was rejected
    __shared__ uint64_t s_Sp, s_Zl;
    __shared__ uint64_t s_U[16], s_Ufin;         // the layer's uniforms
    __shared__ u128 s_F, s_Zrem, s_tt;
    __shared__ float s_M;
    __shared__ int s_ok, s_miss;

    const int tid = threadIdx.x;
    const int lane = tid % WAVE, wid = tid / WAVE;
    // team layout: all G blocks of a sequence on the same XCD
    const int x = blockIdx.x;
    const int G = a.G;
    int b, g;
    {
        const int xcd = x % 8, local = x / 8;
        const int teams_per_xcd = (t.B + 7) / 8;
        b = xcd + 8 * (local / G);
        g = local % G;
        if (local / G >= teams_per_xcd || b >= t.B) return;  // padding blocks
    }
    const int V = t.V, K = t.K, NN = t.NN;
    const int NC = (V + CH - 1) / CH;
    const int64_t nb = (int64_t)b * NN;
    uint64_t* flags = t.team_flag + (int64_t)b * GMAX;
    // this block's ticket: the launch number for the team, ticket / G
    uint64_t ticket = 0;
    if (tid == 0)
        ticket = __hip_atomic_fetch_add(&t.team_ticket[b], 1ull, __ATOMIC_RELAXED,
                                        __HIP_MEMORY_SCOPE_AGENT);
    uint64_t* tmax_x = t.team_max + (int64_t)b * GMAX;
    uint64_t* chunk_x = t.team_chunk + (int64_t)b * NCMAX;
    uint64_t* tsum_x = t.team_sum + (int64_t)b * GMAX;
    uint64_t* nchunk_x = t.team_nchunk + (int64_t)b * NCMAX * 2;   // dense residual totals
    auto nchunk_at = [&](int c) -> u128 {
        const uint64_t lo = __hip_atomic_load(&nchunk_x[2 * c], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const uint64_t hi = __hip_atomic_load(&nchunk_x[2 * c + 1], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return ((u128)hi << 64) | lo;
    };
    const int c0 = g * SEGCH;                 // first chunk of this segment
    const int c1 = min(NC, c0 + SEGCH);

    // the root: pruned index 0; its first child and expanded index
    __shared__ uint64_t s_epoch;
    if (tid == 0) {
        s_cur = 0;
        s_curp = 0;
        s_fc = t.first_child[nb];
        s_e = t.exp_of[nb];
        // barrier epochs of this launch: a window of 64 above the previous
        // launch's (a walk uses 3 per layer, at most 48)
        s_epoch = 64 * (ticket / (uint64_t)G + 1);
    }
    __syncthreads();
    const uint64_t epoch = s_epoch;
    int level = 0, nacc = 0;
    bool failed = false;                      // a team wait timed out, or no finite target logit
    for (;;) {
        const int cur_p = s_curp, fc = s_fc, e = s_e;
        if (level > t.D || cur_p < 0 || cur_p > a.R) {   // unreachable
            if (tid == 0) atomicOr(t.err, 32);
            break;
        }
        const char* row = (const char*)a.logits + ((int64_t)b * (a.R + 1) + cur_p) * t.stride * ESZ;
        // ---- the node's data, then the segment (registers for the first
        //      JREG chunks of each wave), then the logits of the special
        //      tokens this block owns: all in flight together --------------
        const int nt = (fc >= 0 && !DN) ? t.S - t.m : 0;
        const int64_t tb = ((int64_t)b * t.E + (e >= 0 ? e : 0)) * t.S;
        int sp_id = -1;                      // tail entry tid (sparse)
        uint32_t sp_q = 0;
        if (tid < nt) {
            sp_id = t.tail_id[tb + tid];
            sp_q = t.tail_q[tb + tid];
        }
        bool keep = false;
        int kind = -1, ctok = -1, cpidx = -1, cfc = -1, ce = -1, ctail = -1;
        if (tid < WAVE && fc >= 0 && lane < K) {
            const int64_t o = nb + fc + lane;
            cpidx = t.pidx[o];
            kind = (t.meta[o] >> 16) & 0xFF;
            ctok = t.tok[o];
            cfc = t.first_child[o];
            ce = t.exp_of[o];
            ctail = DN ? -1 : t.tidx[o];        // its place in the stored tail
            keep = cpidx > 0;
        }
        const uint64_t Zq = (fc >= 0) ? t.zq[(int64_t)b * t.E + e] : 1;
        uint4 xr[JREG];
#pragma unroll
        for (int j = 0; j < JREG; ++j) {
            const int c = c0 + wid + NWV * j;
            xr[j] = (c < c1) ? load_vec<DT>(row, c * WAVE + lane, V) : make_uint4(0, 0, 0, 0);
        }
        // the logits of the special tokens: every block reads all of them
        // (each block then has p's weights at them without an exchange)
        float sp_l = 0.0f;                   // logit of this thread's tail token
        if (sp_id >= 0) sp_l = load_logit<DT>(row, sp_id);
        // logit of this lane's child (every child, pruned or kept, so that
        // the leads -- the draft's top tokens, not in a stored tail -- enter
        // the guess of the row maximum)
        float c_l = 0.0f;
        if (ctok >= 0) c_l = load_logit<DT>(row, ctok);
        // dense mode: q~ at this node comes from its draft row (borrowed),
        // the logit of its x_{m+1} and its leads
        const char* drow = nullptr;
        float dref = 0.0f;
        const int nlead = (DN && fc >= 0) ? t.m : 0;
        if (DN && fc >= 0) {
            const int rowi = (level == 0) ? b : b * t.NE + (e - 1 - (level - 1) * t.NE);
            drow = (const char*)a.draft[level] + (int64_t)rowi * t.stride * ESZ;
            dref = t.dref[(int64_t)b * t.E + e];
            if (tid < nlead) s_lead[tid] = t.dleads[((int64_t)b * t.E + e) * 16 + tid];
        }
        // ---- candidates: the kept children in slot order (wave 0), the
        //      layer's uniforms, and the stored tail into LDS ---------------
        if (tid < nt) {
            s_tid[tid] = sp_id;
            s_tq[tid] = sp_q;
        }
        for (int i = tid + NTV; i < nt; i += NTV) {
            s_tid[i] = t.tail_id[tb + i];
            s_tq[i] = t.tail_q[tb + i];
        }
        int cpos = -1;
        if (tid < WAVE) {
            uint32_t cq = 0;
            if (DN && keep) {
                bool lead = false;
                for (int q = 0; q < nlead; ++q)
                    lead |= t.dleads[((int64_t)b * t.E + e) * 16 + q] == ctok;
                cq = lead ? 0u : cweight(load_logit<DT>(drow, ctok), dref, a.kT);
            }
            const uint64_t msk = __ballot(keep);
            const uint64_t smk = __ballot(keep && kind == SAMPLED);
            if (keep) {
                cpos = (int)__builtin_amdgcn_mbcnt_hi(
                    (uint32_t)(msk >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)msk, 0u));
                s_c_uid[cpos] = fc + lane;
                s_c_tok[cpos] = ctok;
                s_c_slot[cpos] = lane + 1;
                s_c_zero[cpos] = 0;
                s_c_q[cpos] = cq;
                s_c_pidx[cpos] = cpidx;
                s_c_fc[cpos] = cfc;
                s_c_e[cpos] = ce;
                s_c_tail[cpos] = ctail;
            }
            if (lane == 0) {
                s_nc = __popcll(msk);
                s_spos = smk ? __popcll(msk & ((smk & (~smk + 1)) - 1)) : -1;
            }
        } else if (wid == 1 && lane <= K + 1) {
            // the layer's draws, one per lane: j = 0 the sampled-token test,
            // j = slot for the candidate tests, then the final sample
            const bool fin = lane == K + 1;
            const uint64_t d = philox_draw(a.rng_key, fin ? P_FINAL : P_VERIFY, (uint64_t)b,
                                           fin ? (uint64_t)level : (uint64_t)(32 * level + lane));
            if (fin) s_Ufin = d;
            else s_U[lane] = d >> 32;
        }
        // Weights of the segment relative to Mw: every chunk's total to the
        // team, the wave's sum returned; *over is set if an element of the
        // thread exceeds Mw.  The tail past V reads as -inf, of weight 0 for
        // a finite Mw, so no element needs a bounds test (which would
        // branch per element and serialise the weights).
        auto seg_weights = [&](float Mw, bool* over) -> uint64_t {
            uint64_t wpart = 0;
            bool ov = false;
#pragma unroll
            for (int j = 0; j < JREG; ++j) {
                const int c = c0 + wid + NWV * j;
                if (c < c1) {
                    const uint4 xv = xr[j];
                    uint64_t sum = 0;
                    float vmx = -INFINITY;
#pragma unroll
                    for (int k = 0; k < VEC; k += 2) {
                        // a pair's weights (each <= 2^30) summed in 32 bits
                        const float la = velem<DT>(xv, k), lb = velem<DT>(xv, k + 1);
                        vmx = fmaxf(vmx, fmaxf(la, lb));
                        sum += (uint64_t)(cweight(la, Mw, a.kT) + cweight(lb, Mw, a.kT));
                    }
                    ov |= vmx > Mw;
                    sum = wave_sum_u64(sum);
                    wpart += sum;
                    if (lane == 0)
                        __hip_atomic_store(&chunk_x[c], sum, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_AGENT);
                }
            }
            for (int c = c0 + wid + NWV * JREG; c < c1; c += NWV) {
                const uint4 xv = load_vec<DT>(row, c * WAVE + lane, V);
                uint64_t sum = 0;
                float vmx = -INFINITY;
#pragma unroll
                for (int k = 0; k < VEC; k += 2) {
                    const float la = velem<DT>(xv, k), lb = velem<DT>(xv, k + 1);
                    vmx = fmaxf(vmx, fmaxf(la, lb));
                    sum += (uint64_t)(cweight(la, Mw, a.kT) + cweight(lb, Mw, a.kT));
                }
                ov |= vmx > Mw;
                sum = wave_sum_u64(sum);
                wpart += sum;
                if (lane == 0)
                    __hip_atomic_store(&chunk_x[c], sum, __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
            }
            *over = ov;
            return wpart;
        };
        float M;
        {
            // ---- 1. the row maximum is guessed as the largest target logit
            //         at the special tokens and the pruned children (all of
            //         them in every block); the segment's weights, chunk
            //         totals and p's weights at the special tokens relative
            //         to the guess in one pass, which also notes any element
            //         above the guess; one exchange carries the sums and
            //         whether any segment exceeds the guess.  The row
            //         maximum is at least the guess, so when no segment
            //         exceeds it, it is the row maximum and every weight is
            //         the one relative to it.  Otherwise, and at
            //         a node that was not expanded (no special tokens), the
            //         maximum is exchanged first and the pass follows.
            auto special_weights = [&](float Mw) {
                if (tid < nt) s_tp[tid] = cweight(sp_l, Mw, a.kT);
                for (int i = tid + NTV; i < nt; i += NTV)
                    s_tp[i] = cweight(load_logit<DT>(row, s_tid[i]), Mw, a.kT);
                if (cpos >= 0) s_tp[nt + cpos] = cweight(c_l, Mw, a.kT);
            };
            // a node that was not expanded has no special tokens: no guess
            bool miss = fc < 0;
            M = -INFINITY;
            if (!miss) {
                float gm = (tid < nt) ? sp_l : -INFINITY;
                for (int i = tid + NTV; i < nt; i += NTV)
                    gm = fmaxf(gm, load_logit<DT>(row, s_tid[i]));
                if (ctok >= 0) gm = fmaxf(gm, c_l);
                gm = block_max<NTV>(gm, s_redf);
                bool over;
                const uint64_t wpart = seg_weights(gm, &over);
                special_weights(gm);
                over = __ballot(over) != 0;
                if (lane == 0) s_red[wid] = over ? kMiss : wpart;
                if (!team_sum_exchange(tsum_x, g, G, epoch + 3 * level + 1, s_red, NWV, a.spin,
                                       t.err, &s_ok, &s_Sp, &s_miss)) {
                    failed = true;
                    break;
                }
                M = gm;
                miss = s_miss != 0;
            }
            if (miss) {
                // (the segment read again: cheaper here than keeping more live)
                float mx = -INFINITY;
                for (int c = c0 + wid; c < c1; c += NWV) {
                    const uint4 xv = load_vec<DT>(row, c * WAVE + lane, V);
#pragma unroll
                    for (int k = 0; k < VEC; ++k) mx = fmaxf(mx, velem<DT>(xv, k));
                }
                mx = block_max<NTV>(mx, s_redf);
                if (!team_max_exchange(tmax_x, g, G, epoch + 3 * level + 2, mx, a.spin, t.err,
                                       &s_ok, &s_M)) {
                    failed = true;
                    break;
                }
                M = s_M;
                bool over;
                const uint64_t wpart = seg_weights(M, &over);
                special_weights(M);
                if (lane == 0) s_red[wid] = wpart;
                if (!team_sum_exchange(tsum_x, g, G, epoch + 3 * level + 3, s_red, NWV, a.spin,
                                       t.err, &s_ok, &s_Sp, &s_miss)) {
                    failed = true;
                    break;
                }
            }
        }
        const int nc = s_nc, spos = s_spos;
        if (!(M > -INFINITY)) {
            // no finite target logit at this node: p is undefined.  Every
            // block of the team holds the same M, so all leave here.
            if (g == 0 && tid == 0) atomicOr(t.err, 512);
            failed = true;
            break;
        }
        // ---- 3. Algorithm 1 at this layer, by wave 0 (the chunk totals and
        //         the special weights from the team, S_p, the tail deficit,
        //         and the decisions of lane 0) ---------------------------------
        uint64_t Sp = 0;
        // The remaining candidates' tests in slot order (Algorithm 1), one
        // lane per candidate in [lo, nc_): lane ci holds N_ci (0 for the
        // sampled child);
        // the residual mass before candidate ci is Zrem less the N of the
        // candidates before it (all rejected if ci is reached), so the
        // first lane whose test passes is the accepted candidate.  Returns
        // its index, or -1 with *zrem reduced by every candidate's N; marks
        // the rejected candidates.  Wave 0 only.
        auto cand_tests = [&](int lo, int nc_, int spos_, u128 Nu, u128* zrem) -> int {
            const bool cand = lane >= lo && lane < nc_ && lane != spos_;
            if (!cand) Nu = 0;
            const u128 before = wave_incl_scan_u128(Nu) - Nu;
            const u128 zr = *zrem - before;
            const uint64_t U = cand ? s_U[s_c_slot[lane]] : 0ull;
            const bool pass = cand && ((u128)(U + 1) * zr <= (Nu << 32));
            const uint64_t pm = __ballot(pass);
            const int first = pm ? (int)__builtin_ctzll(pm) : WAVE;
            if (cand && lane < first) s_c_zero[lane] = 1;
            if (pm) return first;
            *zrem -= wave_sum_u128(Nu);
            return -1;
        };
        if (tid < WAVE) {
            // latency-critical single-wave section: issue ahead of the
            // weight passes of other blocks on this compute unit
            __builtin_amdgcn_s_setprio(3);
            Sp = s_Sp;
            wave_sync();

            // RRSw (App. D.2): the leads -- the candidates before the sampled
            // child -- are tested first, under p; the sampled child is then
            // tested under what remains, of mass Z_l.  Algorithm 1 tests the
            // sampled child first (Z_l = S_p).  Every lane takes the same
            // decisions.
            int mode = (nc == 0) ? 2 : 0;      // 0: candidate tests follow, 1: accepted, 2: final sample
            int next = -1, clo = 0;
            uint64_t Zl = Sp;
            if (t.rrsw && spos > 0) {
                u128 zr = Sp;
                const u128 Np = (lane < spos) ? (u128)s_tp[nt + lane] : (u128)0;
                next = cand_tests(0, spos, -1, Np, &zr);
                if (next >= 0) mode = 1;
                Zl = (uint64_t)zr;
                clo = spos + 1;
            }
            if (mode == 0 && spos >= 0) {
                const int yi = s_c_tail[spos];
                if (!DN && yi < 0 && lane == 0) atomicOr(t.err, 4);
                const uint64_t QY = DN ? (uint64_t)s_c_q[spos] : ((yi >= 0) ? s_tq[yi] : 0);
                const uint64_t PY = s_tp[nt + spos];
                const uint64_t U = s_U[0];
                if ((u128)(U + 1) * QY * Zl <= (((u128)PY * Zq) << 32)) {
                    mode = 1;
                    next = spos;
                }
            }
            const bool resid = spos >= 0 && mode == 0;
            const u128 F = resid ? (u128)Zq : (u128)1;
            // no rejected Y: r = p less rejected leads, mass Z_l.  Sparse
            // rejection: Z_r = Zq Z_l less the sum over the tail of
            // min(P_v Zq, Q_v Z_l).  Dense rejection: the residual totals
            // come from a third pass.
            u128 Zrem = Zl;
            if (resid && !DN) {
                u128 d = 0;
                for (int i = lane; i < nt; i += WAVE) {
                    const u128 pz = (u128)s_tp[i] * Zq, qs = (u128)s_tq[i] * Zl;
                    d += pz < qs ? pz : qs;
                }
                Zrem = (u128)Zq * Zl - wave_sum_u128(d);
            }
            if (mode == 0 && !(DN && resid)) {
                u128 Nu = 0;
                if (lane < nc) {
                    const uint64_t P = s_tp[nt + lane];
                    const int ti = s_c_tail[lane];
                    Nu = F * (u128)P;
                    if (resid && ti >= 0) {
                        const u128 pz = (u128)P * Zq, qs = (u128)s_tq[ti] * Zl;
                        Nu = pz > qs ? pz - qs : (u128)0;
                    }
                }
                next = cand_tests(clo, nc, spos, Nu, &Zrem);
                mode = next >= 0 ? 1 : 2;
            }
            if (lane == 0) {
                s_Sp = Sp;
                s_Zl = Zl;
                s_mode = mode;
                s_resid = resid ? 1 : 0;
                s_F = F;
                s_Zrem = Zrem;
                if (mode == 2) s_tt = mulhi_64x128(s_Ufin, Zrem);
                if (mode == 1) {
                    s_token = s_c_tok[next];
                    s_cur = s_c_uid[next];
                    s_curp = s_c_pidx[next];
                    s_fc = s_c_fc[next];
                    s_e = s_c_e[next];
                }
            }
            __builtin_amdgcn_s_setprio(0);
        }
        __syncthreads();
        Sp = s_Sp;
        const uint64_t Zl = s_Zl;
        const bool residual = s_resid != 0;
        const int nrej = (t.rrsw && residual) ? spos : 0;    // leads rejected before Y
        if (DN && s_mode == 0) {
            // N_v = max(0, P_v Zq - Q_v Z_l) over all of V (Q_v from the draft
            // row, 0 at the leads; P_v = 0 at leads rejected before Y):
            // chunk totals over the segment, exchanged
            for (int c = c0 + wid; c < c1; c += NWV) {
                const uint4 xv = load_vec<DT>(row, c * WAVE + lane, V);
                const uint4 dv = load_vec<DT>(drow, c * WAVE + lane, V);
                u128 sum = 0;
#pragma unroll
                for (int k = 0; k < VEC; ++k) {
                    const int v = (c * WAVE + lane) * VEC + k;
                    if (v < V) {
                        bool lead = false, rej = false;
                        for (int q = 0; q < nlead; ++q) lead |= s_lead[q] == v;
                        for (int q = 0; q < nrej; ++q) rej |= s_c_tok[q] == v;
                        const uint64_t P = rej ? 0u : cweight(velem<DT>(xv, k), M, a.kT);
                        const uint64_t Q = lead ? 0u : cweight(velem<DT>(dv, k), dref, a.kT);
                        const u128 pz = (u128)P * Zq, qs = (u128)Q * Zl;
                        sum += pz > qs ? pz - qs : (u128)0;
                    }
                }
                sum = wave_sum_u128(sum);
                if (lane == 0) {
                    __hip_atomic_store(&nchunk_x[2 * c], (uint64_t)sum, __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
                    __hip_atomic_store(&nchunk_x[2 * c + 1], (uint64_t)(sum >> 64), __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
                }
            }
            if (!team_barrier(flags, g, G, epoch + 3 * level + 3, a.spin, t.err, &s_ok)) {
                failed = true;
                break;
            }
            if (tid < WAVE) {
                __builtin_amdgcn_s_setprio(3);
                u128 part = 0;
                for (int c = lane; c < NC; c += WAVE) part += nchunk_at(c);
                u128 Zrem = wave_sum_u128(part);
                u128 Nu = 0;
                if (lane < nc) {
                    const uint64_t P = s_tp[nt + lane];
                    const u128 pz = (u128)P * Zq, qs = (u128)s_c_q[lane] * Zl;
                    Nu = pz > qs ? pz - qs : (u128)0;
                }
                const int next = cand_tests(t.rrsw ? spos + 1 : 0, nc, spos, Nu, &Zrem);
                if (lane == 0) {
                    s_mode = next >= 0 ? 1 : 2;
                    s_Zrem = Zrem;
                    if (next < 0) s_tt = mulhi_64x128(s_Ufin, Zrem);
                    if (next >= 0) {
                        s_token = s_c_tok[next];
                        s_cur = s_c_uid[next];
                        s_curp = s_c_pidx[next];
                        s_fc = s_c_fc[next];
                        s_e = s_c_e[next];
                    }
                }
                __builtin_amdgcn_s_setprio(0);
            }
            __syncthreads();
        }
        if (s_mode == 1) {
            if (g == 0 && tid == 0) a.accepted[(int64_t)b * t.D + nacc] = s_token;
            ++nacc;
            ++level;
            __syncthreads();
            continue;
        }
        // ---- final sample u* ~ r (one block of the team) --------------------
        if (g != 0) break;
        {
            // the chunk totals, published before the sum exchange; for
            // the residual, every chunk's sum of min(P_v Zq, Q_v Z_l) over
            // the live tail tokens in it, gathered from the tail entries in
            // two limbs: the deficit is below 2^71 (P_v <= 2^30, Zq < 2^40),
            // so its low 40 bits and the rest (< 2^31), summed over at most
            // 1023 entries, stay below 2^64
            for (int c = tid; c < NC; c += NTV) {
                s_chunk[c] = __hip_atomic_load(&chunk_x[c], __ATOMIC_RELAXED,
                                               __HIP_MEMORY_SCOPE_AGENT);
                s_dlo[c] = 0;
                s_dhi[c] = 0;
            }
            __syncthreads();
            if (residual) {
                for (int i = tid; i < nt; i += NTV) {
                    const u128 pz = (u128)s_tp[i] * Zq, qs = (u128)s_tq[i] * Zl;
                    const u128 d = pz < qs ? pz : qs;
                    const int c = s_tid[i] / CH;
                    atomicAdd(&s_dlo[c], (uint64_t)d & ((1ull << 40) - 1));
                    atomicAdd(&s_dhi[c], (uint64_t)(d >> 40));
                }
                __syncthreads();
            }
        }
        const u128 F = s_F;
        const u128 tt = s_tt;
        // corrected chunk totals, contiguous chunk ranges per thread
        const int cpt = (NC + NTV - 1) / NTV;
        const int ca = min(NC, tid * cpt), cz = min(NC, ca + cpt);
        auto special_def = [&](int cidx, u128* def_out) {
            // F * P_v - N_v summed over the special tokens of chunk cidx
            u128 d = 0;
            // the live tail tokens (sparse), gathered per chunk above
            if (!DN && residual) d = (u128)s_dlo[cidx] + ((u128)s_dhi[cidx] << 40);
            for (int ci = 0; ci < nc; ++ci) {
                if (!s_c_zero[ci]) continue;
                const int v = s_c_tok[ci];
                if (v / CH != cidx) continue;
                const u128 fp = F * (u128)s_tp[nt + ci];
                if (residual && s_c_tail[ci] >= 0) {
                    // zeroed tail token: its live deficit was counted above
                    const u128 pz = (u128)s_tp[nt + ci] * Zq, qs = (u128)s_tq[s_c_tail[ci]] * Zl;
                    d += fp - (pz < qs ? pz : qs);
                } else {
                    d += fp;
                }
            }
            *def_out = d;
        };
        // chunk weight of r: dense residual totals, else F times p's chunk
        // total, less the special tokens' corrections
        auto chunk_w = [&](int c) -> u128 {
            if (DN && residual) {
                u128 w = nchunk_at(c);
                for (int ci = 0; ci < nc; ++ci) {
                    // (rejected leads were left out of the third pass)
                    if (!s_c_zero[ci] || ci < nrej || s_c_tok[ci] / CH != c) continue;
                    const u128 pz = (u128)s_tp[nt + ci] * Zq, qs = (u128)s_c_q[ci] * Zl;
                    w -= pz > qs ? pz - qs : (u128)0;
                }
                return w;
            }
            u128 d;
            special_def(c, &d);
            return F * (u128)s_chunk[c] - d;
        };
        u128 mysum = 0;
        for (int c = ca; c < cz; ++c) mysum += chunk_w(c);
        u128 total;
        const u128 pre = block_excl_scan_u128(mysum, s_w128, &total);
        if (tid == 0) s_cstar = -1;
        __syncthreads();
        if (tt >= pre && tt < pre + mysum) {
            u128 acc = pre;
            for (int c = ca; c < cz; ++c) {
                const u128 w = (cz - ca == 1) ? mysum : chunk_w(c);   // (one chunk: known)
                if (tt < acc + w) {
                    s_cstar = c;
                    s_tt = tt - acc;
                    break;
                }
                acc += w;
            }
        }
        __syncthreads();
        const int cs = s_cstar;
        if (cs < 0) {
            if (tid == 0) atomicOr(t.err, 8);
            break;
        }
        // scan of chunk cs: F * P for every token, then the special tokens
        // (live tail tokens get their residual weight, zeroed candidates 0),
        // then a block scan
        const u128 t2 = s_tt;
        for (int i = tid; i < CH; i += NTV) {
            const int v = cs * CH + i;
            u128 w = 0;
            if (v < V) {
                const uint64_t P = cweight(load_logit<DT>(row, v), M, a.kT);
                if (DN && residual) {
                    bool lead = false;
                    for (int q = 0; q < nlead; ++q) lead |= s_lead[q] == v;
                    const uint64_t Q = lead ? 0u : cweight(load_logit<DT>(drow, v), dref, a.kT);
                    const u128 pz = (u128)P * Zq, qs = (u128)Q * Zl;
                    w = pz > qs ? pz - qs : (u128)0;
                } else {
                    w = F * (u128)P;
                }
            }
            s_cn[i] = w;
        }
        __syncthreads();
        if (residual) {
            for (int i = tid; i < nt; i += NTV) {
                const int v = s_tid[i];
                if (v / CH == cs) {
                    const u128 pz = (u128)s_tp[i] * Zq, qs = (u128)s_tq[i] * Zl;
                    s_cn[v - cs * CH] = pz > qs ? pz - qs : (u128)0;
                }
            }
        }
        __syncthreads();
        if (tid < nc && s_c_zero[tid] && s_c_tok[tid] / CH == cs) s_cn[s_c_tok[tid] - cs * CH] = 0;
        __syncthreads();
        constexpr int TPT = CH / NTV;          // tokens per thread (1 or 2)
        u128 mine = 0;
#pragma unroll
        for (int q = 0; q < TPT; ++q) mine += s_cn[tid * TPT + q];
        const u128 pre2 = block_excl_scan_u128(mine, s_w128, &total);
        if (tid == 0) s_token = -1;
        __syncthreads();
        if (t2 >= pre2 && t2 < pre2 + mine) {
            u128 acc = pre2;
#pragma unroll
            for (int q = 0; q < TPT; ++q) {
                acc += s_cn[tid * TPT + q];
                if (t2 < acc) {
                    s_token = cs * CH + tid * TPT + q;
                    break;
                }
            }
        }
        __syncthreads();
        if (tid == 0) {
            const int tok = s_token;
            if (tok < 0) atomicOr(t.err, 8);
            a.final_token[b] = tok;
            a.accept_len[b] = nacc;
            for (int i = nacc; i < t.D; ++i) a.accepted[(int64_t)b * t.D + i] = -1;
        }
        break;
    }
    // a timed-out wait or an undefined target row: the walk did not
    // complete, so the team's first block (the only one that writes outputs)
    // reports a defined failure instead
    if (failed && g == 0 && tid == 0) {
        a.accept_len[b] = -1;
        a.final_token[b] = -1;
        for (int i = 0; i < t.D; ++i) a.accepted[(int64_t)b * t.D + i] = -1;
    }
}

static const void* verify_fn(const TreeDev& t) {
    if (t.dense) return t.dtype ? (const void*)&k_verify<1, 1> : (const void*)&k_verify<0, 1>;
    return t.dtype ? (const void*)&k_verify<1, 0> : (const void*)&k_verify<0, 0>;
}

// Team shape for a tree: about `target` blocks in all (1024 by default),
// segments of whole chunks, G <= GMAX, and no more blocks than the device
// holds at once, so every block can be resident together.
hipError_t verify_shape(const TreeDev& t, int* G_out, int* segch, int* grid) {
    const int VEC = t.dtype ? 8 : 4;
    const int NC = (t.V + WAVE * VEC - 1) / (WAVE * VEC);
    const char* env = getenv("RHEO_VERIFY_BLOCKS");
    const int target = env ? atoi(env) : 1024;
    int dev = 0, cus = 0, per_cu = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    const void* fn = verify_fn(t);
    if (e == hipSuccess) e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, NTV, 0);
    if (e != hipSuccess) return e;
    const int teams_per_xcd = (t.B + 7) / 8;
    int G = target / (8 * teams_per_xcd);
    if (G > GMAX) G = GMAX;
    if (G > NC) G = NC;
    while (G > 1 && 8 * teams_per_xcd * G > per_cu * cus) --G;
    if (G < 1) G = 1;
    const int blocks = 8 * teams_per_xcd * G;
    if (blocks > per_cu * cus) return hipErrorCooperativeLaunchTooLarge;
    *G_out = G;
    *segch = (NC + G - 1) / G;
    *grid = blocks;
    return hipSuccess;
}

// The grid never exceeds what the device holds at once (verify_shape), so
// on a device that runs nothing else every block is resident from the
// start and the team barriers complete; a barrier that waits past its spin
// limit, because other work held part of the device, ends the walk with the
// failure result and device error 128 rather than hanging.
hipError_t launch_verify(const TreeDev& t, const VerifyArgs& a, int segch, int grid,
                         hipStream_t s) {
    const void* fn = verify_fn(t);
    TreeDev tt = t;
    VerifyArgs aa = a;
    aa.NV = segch;
    void* args[] = {&tt, &aa};
    return hipLaunchKernel(fn, dim3(grid), dim3(NTV), args, 0, s);
}

}  // namespace rheo
