// Device-side building blocks of the RheoSampling hot path (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rheo {

typedef unsigned __int128 u128;

constexpr int WAVE = 64;

enum Kind { LEAD = 0, SAMPLED = 1, FILL = 2 };
enum Purpose { P_DRAFT = 1, P_VERIFY = 2, P_FINAL = 3 };

// ---------------------------------------------------------------------------
// Philox4x64-10 (Salmon, Moraes, Dror, Shaw, SC'11): ten rounds of two
// 64x64->128 multiplies with the round multipliers, the high halves xored
// into the odd words with the key, key bumped by the Weyl constants.
// ---------------------------------------------------------------------------
__device__ inline uint64_t philox_draw(uint64_t key, uint64_t purpose,
                                       uint64_t seq, uint64_t index) {
    uint64_t x0 = index, x1 = seq, x2 = purpose, x3 = 0;
    uint64_t k0 = key, k1 = 0;
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        if (r) {
            k0 += 0x9E3779B97F4A7C15ull;
            k1 += 0xBB67AE8584CAA73Bull;
        }
        const uint64_t lo0 = 0xD2E7470EE14C6C93ull * x0;
        const uint64_t hi0 = __umul64hi(0xD2E7470EE14C6C93ull, x0);
        const uint64_t lo1 = 0xCA5A826395121157ull * x2;
        const uint64_t hi1 = __umul64hi(0xCA5A826395121157ull, x2);
        const uint64_t n0 = hi1 ^ x1 ^ k0;
        const uint64_t n2 = hi0 ^ x3 ^ k1;
        x0 = n0; x1 = lo1; x2 = n2; x3 = lo0;
    }
    return x0;
}

// ---------------------------------------------------------------------------
// Canonical integer weight of a logit: floor(2^30 * 2^t) with
// t = fl(fl(l - ref) * kT), kT = fl32(log2(e) / T), t clamped to <= 0 and
// weight 0 below t = -31.  2^t = 2^n * P(f), n = rint(t), f = t - n, P the
// degree-6 Taylor polynomial of 2^f with coefficients (ln 2)^k / k! * 2^30
// rounded to fp32, evaluated in Horner form, each step one fused
// multiply-add (v_fma_f32: a single rounding).  Result: floor(2^30 P 2^n) =
// (uint32)(2^30 P) >> -n,
// taken as the truncating conversion of the exact product 2^30 P * 2^n
// (a scaling by a power of two, exact; below t = -31 it is < 1, so 0).
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t cweight_of_t(float t) {
    const float n = rintf(t);
    const float f = __fsub_rn(t, n);
    float p = 0x1.430912p+17f;
    p = __fmaf_rn(p, f, 0x1.5d87fep+20f);
    p = __fmaf_rn(p, f, 0x1.3b2ab6p+23f);
    p = __fmaf_rn(p, f, 0x1.c6b08ep+25f);
    p = __fmaf_rn(p, f, 0x1.ebfbe0p+27f);
    p = __fmaf_rn(p, f, 0x1.62e430p+29f);
    p = __fmaf_rn(p, f, 0x1.000000p+30f);
    return (uint32_t)__builtin_amdgcn_ldexpf(p, (int)n);
}
__device__ __forceinline__ uint32_t cweight(float l, float ref, float kT) {
    const float t = __fmul_rn(__fsub_rn(l, ref), kT);
    // t clamped to [-64, 0] in one instruction (t is never NaN for a finite
    // ref; a signed zero may come out either way, of the same weight)
    return cweight_of_t(__builtin_amdgcn_fmed3f(t, -64.0f, 0.0f));
}
// The same weight for l <= ref (then t <= 0 and the upper clamp is void).
__device__ __forceinline__ uint32_t cweight_below(float l, float ref, float kT) {
    const float t = __fmul_rn(__fsub_rn(l, ref), kT);
    return cweight_of_t(fmaxf(t, -64.0f));
}

// Order-preserving map of an fp32 value to uint32 (-0 folded onto +0).
__device__ __forceinline__ uint32_t ord32(float f) {
    uint32_t b = __float_as_uint(f);
    if (b == 0x80000000u) b = 0u;
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}
__device__ __forceinline__ float unord32(uint32_t k) {
    const uint32_t b = (k & 0x80000000u) ? (k & 0x7fffffffu) : ~k;
    return __uint_as_float(b);
}
// Selection key of a logit: larger key = (larger logit, then smaller id).
__device__ __forceinline__ uint64_t logit_key(float v, uint32_t id) {
    return ((uint64_t)ord32(v) << 32) | (uint64_t)(0xFFFFFFFFu - id);
}
__device__ __forceinline__ float key_value(uint64_t k) { return unord32((uint32_t)(k >> 32)); }
__device__ __forceinline__ int key_id(uint64_t k) { return (int)(0xFFFFFFFFu - (uint32_t)k); }

// Priority of a tree node (App. C.1): score descending, depth ascending,
// slot path ascending -- as a 128-bit key where larger = better.  Scores
// are non-negative, so their IEEE bits are already order-preserving.
__device__ __forceinline__ void prio_key(double score, int depth, uint64_t path,
                                         uint64_t& hi, uint64_t& lo) {
    hi = (uint64_t)__double_as_longlong(score);
    lo = ((uint64_t)(15 - depth) << 60) | (0x0FFFFFFFFFFFFFFFull - path);
}

// 16-byte streaming load (non-temporal: the row is read once).
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 load_stream16(const void* p) {
    const u32x4 v = __builtin_nontemporal_load((const u32x4*)p);
    return make_uint4(v.x, v.y, v.z, v.w);
}

// Clears the IEEE bit of the wave's MODE register (hardware register 1,
// bit 9).  With it clear, v_max_f32 / v_max3_f32 return the other operand
// of a NaN operand, signalling or quiet, instead of quieting it.  Kernels
// that take maxima over raw bf16-pair words call it first: such a word is a
// NaN whenever its high element is -inf and its low element is not +0, and
// row padding is a NaN pattern, so both must drop out of the maxima.  It
// changes nothing for non-NaN operands.
__device__ __forceinline__ void ieee_mode_off() { __builtin_amdgcn_s_setreg(1 | (9 << 6), 0); }

// bf16 pairs packed in a uint32: low and high element as fp32 (exact).
__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// High 128 bits of a (64 x 128)-bit product, b < 2^96.
__device__ __forceinline__ u128 mulhi_64x128(uint64_t a, u128 b) {
    const uint64_t blo = (uint64_t)b;
    const uint64_t bhi = (uint64_t)(b >> 64);
    const u128 plo = (u128)a * blo;
    return (u128)a * bhi + (plo >> 64);
}

// ---------------------------------------------------------------------------
// wave / block reductions (wave64)
// ---------------------------------------------------------------------------
// Lane movement inside rows of 16 lanes (DPP): rotate right by N, and shift
// right by N with zeros shifted in.  Reductions and scans built on them stay
// in the vector ALU (no LDS round trip); all 64 lanes must be active.
template <int N>
__device__ __forceinline__ uint32_t row_ror(uint32_t v) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x120 + N, 0xF, 0xF, false);
}
template <int N>
__device__ __forceinline__ uint32_t row_shr(uint32_t v) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x110 + N, 0xF, 0xF, true);
}
template <int N>
__device__ __forceinline__ uint64_t row_ror64(uint64_t v) {
    return ((uint64_t)row_ror<N>((uint32_t)(v >> 32)) << 32) | row_ror<N>((uint32_t)v);
}
template <int N>
__device__ __forceinline__ uint64_t row_shr64(uint64_t v) {
    return ((uint64_t)row_shr<N>((uint32_t)(v >> 32)) << 32) | row_shr<N>((uint32_t)v);
}
// Orders LDS accesses of the lanes of one wave (no block barrier).
__device__ __forceinline__ void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
}
__device__ __forceinline__ uint32_t lane_u32(uint32_t v, int l) {
    return (uint32_t)__builtin_amdgcn_readlane((int)v, l);
}
__device__ __forceinline__ uint64_t lane_u64(uint64_t v, int l) {
    return ((uint64_t)lane_u32((uint32_t)(v >> 32), l) << 32) | lane_u32((uint32_t)v, l);
}

__device__ __forceinline__ float wave_max(float v) {
    uint32_t x = __float_as_uint(v);
    x = __float_as_uint(fmaxf(__uint_as_float(x), __uint_as_float(row_ror<8>(x))));
    x = __float_as_uint(fmaxf(__uint_as_float(x), __uint_as_float(row_ror<4>(x))));
    x = __float_as_uint(fmaxf(__uint_as_float(x), __uint_as_float(row_ror<2>(x))));
    x = __float_as_uint(fmaxf(__uint_as_float(x), __uint_as_float(row_ror<1>(x))));
    return fmaxf(fmaxf(__uint_as_float(lane_u32(x, 0)), __uint_as_float(lane_u32(x, 16))),
                 fmaxf(__uint_as_float(lane_u32(x, 32)), __uint_as_float(lane_u32(x, 48))));
}
__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) {
    v += row_ror64<8>(v);
    v += row_ror64<4>(v);
    v += row_ror64<2>(v);
    v += row_ror64<1>(v);
    return lane_u64(v, 0) + lane_u64(v, 16) + lane_u64(v, 32) + lane_u64(v, 48);
}
__device__ __forceinline__ int wave_sum_i32(int v) {
    uint32_t x = (uint32_t)v;
    x += row_ror<8>(x);
    x += row_ror<4>(x);
    x += row_ror<2>(x);
    x += row_ror<1>(x);
    return (int)(lane_u32(x, 0) + lane_u32(x, 16) + lane_u32(x, 32) + lane_u32(x, 48));
}

template <int NT>
__device__ float block_max(float v, float* sh) {
    v = wave_max(v);
    const int w = threadIdx.x / WAVE, l = threadIdx.x % WAVE;
    __syncthreads();
    if (l == 0) sh[w] = v;
    __syncthreads();
    float r = sh[0];
#pragma unroll
    for (int i = 1; i < NT / WAVE; ++i) r = fmaxf(r, sh[i]);
    return r;
}

template <int NT>
__device__ uint64_t block_sum_u64(uint64_t v, uint64_t* sh) {
    v = wave_sum_u64(v);
    const int w = threadIdx.x / WAVE, l = threadIdx.x % WAVE;
    __syncthreads();
    if (l == 0) sh[w] = v;
    __syncthreads();
    uint64_t r = 0;
#pragma unroll
    for (int i = 0; i < NT / WAVE; ++i) r += sh[i];
    return r;
}

// Two block sums in one exchange; sh holds 2 * NT / WAVE words.
template <int NT>
__device__ void block_sum2_u64(uint64_t a, uint64_t b, uint64_t* sh, uint64_t* ra, uint64_t* rb) {
    constexpr int NW = NT / WAVE;
    a = wave_sum_u64(a);
    b = wave_sum_u64(b);
    const int w = threadIdx.x / WAVE, l = threadIdx.x % WAVE;
    __syncthreads();
    if (l == 0) {
        sh[w] = a;
        sh[NW + w] = b;
    }
    __syncthreads();
    uint64_t x = 0, y = 0;
#pragma unroll
    for (int i = 0; i < NW; ++i) {
        x += sh[i];
        y += sh[NW + i];
    }
    *ra = x;
    *rb = y;
}

template <int NT>
__device__ int block_sum_i32(int v, int* sh) {
    v = wave_sum_i32(v);
    const int w = threadIdx.x / WAVE, l = threadIdx.x % WAVE;
    __syncthreads();
    if (l == 0) sh[w] = v;
    __syncthreads();
    int r = 0;
#pragma unroll
    for (int i = 0; i < NT / WAVE; ++i) r += sh[i];
    return r;
}

// Exclusive prefix of v over the wave (lane order).
__device__ __forceinline__ int wave_excl_scan(int v) {
    const int row = (threadIdx.x % WAVE) >> 4;
    uint32_t x = (uint32_t)v;
    x += row_shr<1>(x);
    x += row_shr<2>(x);
    x += row_shr<4>(x);
    x += row_shr<8>(x);
    const uint32_t r0 = lane_u32(x, 15), r1 = lane_u32(x, 31), r2 = lane_u32(x, 47);
    x += (row >= 1 ? r0 : 0u) + (row >= 2 ? r1 : 0u) + (row >= 3 ? r2 : 0u);
    return (int)x - v;
}

}  // namespace rheo

namespace rheo {

// Wave-wide inclusive prefix sum of 64-bit values.
__device__ __forceinline__ uint64_t wave_incl_scan_u64(uint64_t v) {
    const int row = (threadIdx.x % WAVE) >> 4;
    v += row_shr64<1>(v);
    v += row_shr64<2>(v);
    v += row_shr64<4>(v);
    v += row_shr64<8>(v);
    const uint64_t r0 = lane_u64(v, 15), r1 = lane_u64(v, 31), r2 = lane_u64(v, 47);
    v += (row >= 1 ? r0 : 0ull) + (row >= 2 ? r1 : 0ull) + (row >= 3 ? r2 : 0ull);
    return v;
}

// Block-wide exclusive prefix sum of 64-bit values (one value per thread);
// sh holds NT / WAVE words.  Also returns the total through *total.
template <int NT>
__device__ uint64_t block_excl_scan_u64(uint64_t v, uint64_t* sh, uint64_t* total) {
    const int w = threadIdx.x / WAVE, l = threadIdx.x % WAVE;
    const uint64_t inc = wave_incl_scan_u64(v);
    __syncthreads();
    if (l == WAVE - 1) sh[w] = inc;
    __syncthreads();
    uint64_t base = 0, tot = 0;
#pragma unroll
    for (int i = 0; i < NT / WAVE; ++i) {
        if (i < w) base += sh[i];
        tot += sh[i];
    }
    *total = tot;
    return base + inc - v;
}

// Descending bitonic sort of one float per lane across a wave.
__device__ __forceinline__ float wave_sort_desc(float v) {
    const int lane = threadIdx.x % WAVE;
#pragma unroll
    for (int k = 2; k <= WAVE; k <<= 1) {
#pragma unroll
        for (int j = k >> 1; j > 0; j >>= 1) {
            const float o = __shfl_xor(v, j);
            const bool take_max = ((lane & j) == 0) == ((lane & k) == 0);
            v = take_max ? fmaxf(v, o) : fminf(v, o);
        }
    }
    return v;
}

// rank[i] = number of keys strictly greater than keys[i], for unique keys
// in LDS; each key is compared by a group of F consecutive lanes.  With
// `out`, the lane that finishes key i writes it to out[rank] instead when
// the rank is below nsel (and writes no rank), so no barrier is needed
// between ranking and placing.
template <int NT>
__device__ void rank_keys(const uint64_t* keys, int n, int16_t* rank, uint64_t* out = nullptr,
                          int nsel = 0) {
    int npad = 1;
    while (npad < n) npad <<= 1;
    int F = NT / npad;
    if (F < 1) F = 1;
    if (F > WAVE) F = WAVE;
    const int sub = threadIdx.x % F;
    const int per = NT / F;
    // lane `sub` of a key's F lanes compares it with keys [j0, j1), a run of
    // even length and start, read two at a time (keys are 16-byte aligned)
    const int L = ((n + F - 1) / F + 1) & ~1;
    const int j0 = min(sub * L, n), j1 = min(j0 + L, n);
    const ulonglong2* kp = (const ulonglong2*)keys;
    for (int base = 0; base < n; base += per) {
        const int i = base + threadIdx.x / F;
        int cnt = 0;
        if (i < n) {
            const uint64_t k = keys[i];
            int j = j0;
            for (; j + 7 < j1; j += 8) {
                const ulonglong2 a = kp[j / 2], b = kp[j / 2 + 1], c = kp[j / 2 + 2],
                                 d = kp[j / 2 + 3];
                cnt += (a.x > k) + (a.y > k) + (b.x > k) + (b.y > k) + (c.x > k) + (c.y > k) +
                       (d.x > k) + (d.y > k);
            }
            for (; j + 1 < j1; j += 2) {
                const ulonglong2 a = kp[j / 2];
                cnt += (a.x > k) + (a.y > k);
            }
            if (j < j1) cnt += keys[j] > k;
        }
        for (int o = 1; o < F; o <<= 1) cnt += __shfl_xor(cnt, o);
        if (i < n && sub == 0) {
            if (out) {
                if (cnt < nsel) out[cnt] = keys[i];
            } else {
                rank[i] = (int16_t)cnt;
            }
        }
    }
}

// rank[i] = number of 128-bit keys strictly greater than key i (unique keys
// in LDS as {hi, lo} pairs).  One key per lane; every lane of a wave reads
// the same key at the same time (LDS broadcast).
template <int NT>
__device__ void rank_keys128(const ulonglong2* keys, int n, int16_t* rank) {
    for (int base = 0; base < n; base += NT) {
        const int i = base + threadIdx.x;
        const ulonglong2 k = keys[i < n ? i : 0];
        int cnt = 0;
#pragma unroll 8
        for (int j = 0; j < n; ++j) {
            const ulonglong2 x = keys[j];
            cnt += (int)(x.x > k.x) | ((int)(x.x == k.x) & (int)(x.y > k.y));
        }
        if (i < n) rank[i] = (int16_t)cnt;
    }
}

// Hides register-resident 16-byte vectors from the optimiser between
// passes, so each pass unpacks bf16 pairs on the fly instead of keeping
// every element unpacked across the whole kernel.
template <int NV>
__device__ __forceinline__ void opaque_regs(uint4 (&r)[NV]) {
#pragma unroll
    for (int i = 0; i < NV; ++i)
        asm volatile("" : "+v"(r[i].x), "+v"(r[i].y), "+v"(r[i].z), "+v"(r[i].w));
}

}  // namespace rheo
