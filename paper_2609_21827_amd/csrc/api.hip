// Host side of the C ABI declared in include/rheo.h: validation, device
// state, step order and kernel launches.  Nothing here synchronises except
// rheo_destroy and rheo_device_error.
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>

#include <mutex>

#include "rheo.h"
#include "rheo_state.h"

using namespace rheo;

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}

int hip_fail(hipError_t e, const char* what) {
    return fail(RHEO_EHIP, "%s: %s", what, hipGetErrorString(e));
}

enum State { CREATED, EXPANDING, EXPANDED, PRUNED, VERIFIED };

constexpr int kMaxV = 262143;

float k_of_T(float T) { return (float)(1.4426950408889634 / (double)T); }

// tokens of one 64-vector sub-chunk (16-byte vectors of bf16 or fp32)
// Rows in a level from which the per-row kernel runs (it is the faster of
// the two at every level size measured, down to a single row).
constexpr int kRowMin = 1;

int WAVE_TOKENS(int dtype) { return 64 * (dtype == RHEO_BF16 ? 8 : 4); }

// A chunk size fits when the row's chunk lists fit the merge (and, in dense
// mode, the weights pass's copy of them).
bool variant_fits(int dtype, int v, int V, int SL, bool dense) {
    const ExpandVariant ev = expand_variant(dtype, v, V, SL);
    return ev.ok && (!dense || ev.C * ev.Sc <= 512);
}

}  // namespace

struct rheo_tree {
    rheo_config cfg;
    TreeDev dev;
    State state = CREATED;
    int level = 0;
    int R = 0;
    int variant = 0;
    int row_mode = 0;                     // sparse levels: 1 one block per row, 0 chunks,
                                          // -1 by the number of rows
    int vG = 1, v_segch = 1, v_grid = 1;  // verification team shape
    int row_min = kRowMin;                // fewest rows for the per-row kernel
    float T_step = 1.0f;                  // temperature and key of the current step
    uint64_t key_step = 0;
    void* blocks[48] = {};
    const void* draft[16] = {};           // dense: each level's draft rows (borrowed)
    int nblocks = 0;
    bool is_static = false;               // device state in the static scratch array
};

namespace {

template <typename T>
int dalloc(rheo_tree* t, T** p, size_t count) {
    const size_t bytes = count * sizeof(T) ? count * sizeof(T) : 16;
    void* q = nullptr;
    const hipError_t e = hipMalloc(&q, bytes);
    if (e != hipSuccess) return fail(RHEO_ENOMEM, "hipMalloc(%zu): %s", bytes, hipGetErrorString(e));
    t->blocks[t->nblocks++] = q;
    *p = (T*)q;
    return RHEO_OK;
}

void free_all(rheo_tree* t) {
    for (int i = 0; i < t->nblocks; ++i) (void)hipFree(t->blocks[i]);
    t->nblocks = 0;
}

int check_ptr(const void* p, const char* name) {
    if (!p) return fail(RHEO_EINVAL, "%s is NULL", name);
    if ((uintptr_t)p % 16) return fail(RHEO_EINVAL, "%s is not 16-byte aligned", name);
    return RHEO_OK;
}

int check_T(float T) {
    if (!(T > 0.0f) || !std::isfinite(T)) return fail(RHEO_EINVAL, "temperature must be finite and > 0");
    if (!std::isfinite(k_of_T(T))) return fail(RHEO_EINVAL, "temperature too small");
    return RHEO_OK;
}

// Every call of one step takes the step's temperature and key: the stored
// tail weights (and, in dense mode, the q~ verification recomputes from the
// draft rows) and the draws of the sampled slots depend on both.
int check_step_args(const rheo_tree* t, float T, uint64_t key, const char* call) {
    if (std::memcmp(&T, &t->T_step, sizeof(float)) != 0 || key != t->key_step)
        return fail(RHEO_EINVAL, "%s: T and rng_key must be those of the step's first "
                    "rheo_expand_level", call);
    return RHEO_OK;
}

// Validates cfg and fills the handle's host fields (no device work).
int configure(const rheo_config* cfg_in, rheo_tree* t) {
    if (!cfg_in) return fail(RHEO_EINVAL, "NULL argument");
    rheo_config c = *cfg_in;
    if (c.n_expand == 0) c.n_expand = c.pool;
    if (c.eps_m0 == 0.0) c.eps_m0 = std::ldexp(1.0, -40);
    if (c.batch < 1) return fail(RHEO_EINVAL, "batch must be >= 1");
    if (c.vocab < 2 || c.vocab > kMaxV) return fail(RHEO_EINVAL, "vocab must be in [2, %d]", kMaxV);
    if (c.pool < 1 || c.pool > 15) return fail(RHEO_EINVAL, "pool K must be in [1, 15]");
    if (c.leads < 0 || c.leads > c.pool - 1) return fail(RHEO_EINVAL, "leads m must be in [0, K-1]");
    if (c.depth < 1 || c.depth > 15) return fail(RHEO_EINVAL, "depth must be in [1, 15]");
    if (c.n_expand < 1 || c.n_expand > c.pool) return fail(RHEO_EINVAL, "n_expand must be in [1, K]");
    if (c.dtype != RHEO_F32 && c.dtype != RHEO_BF16) return fail(RHEO_EINVAL, "unknown dtype");
    if (c.method < RHEO_METHOD_RHEO || c.method > RHEO_METHOD_TOPK)
        return fail(RHEO_EINVAL, "unknown method %d", c.method);
    if (c.construct_full != 0 && c.construct_full != 1)
        return fail(RHEO_EINVAL, "construct_full must be 0 or 1");
    // support <= 0: dense mode, the support is the whole vocabulary
    const bool dense = c.support <= 0;
    const int S = dense ? c.vocab : (c.support < c.vocab ? c.support : c.vocab);
    if (c.pool > c.vocab) return fail(RHEO_EINVAL, "pool K must be <= vocab");
    if (S < c.pool) return fail(RHEO_EINVAL, "support must be >= pool K");
    if (!dense && S > 1024) return fail(RHEO_EINVAL, "support must be <= 1024");
    if (S <= c.leads) return fail(RHEO_EINVAL, "support must exceed leads m");
    // list length of the selection pass: the support, or in dense mode the
    // m + K tokens the pool can use
    const int SL = dense ? (c.vocab < c.leads + c.pool ? c.vocab : c.leads + c.pool) : S;
    if (c.row_stride < c.vocab) return fail(RHEO_EINVAL, "row_stride must be >= vocab");
    const int esz = c.dtype == RHEO_BF16 ? 2 : 4;
    if ((c.row_stride * esz) % 16) return fail(RHEO_EINVAL, "row_stride must be a multiple of 16 bytes");
    if (!(c.eps_m0 > 0.0) || !std::isfinite(c.eps_m0)) return fail(RHEO_EINVAL, "eps_m0 must be > 0");

    t->cfg = c;
    TreeDev& d = t->dev;
    d.B = c.batch; d.V = c.vocab; d.K = c.pool; d.m = c.leads; d.D = c.depth;
    d.NE = c.n_expand; d.S = S; d.dtype = c.dtype; d.stride = c.row_stride;
    d.rrsw = c.method == RHEO_METHOD_RRSW;
    d.topk = c.method == RHEO_METHOD_TOPK;
    d.dense = dense ? 1 : 0;
    // a support of the whole vocabulary already constructs over all of it
    d.cfull = (!dense && c.construct_full && S < c.vocab) ? 1 : 0;
    d.NCH = (c.vocab + WAVE_TOKENS(c.dtype) - 1) / WAVE_TOKENS(c.dtype);
    d.eps = c.eps_m0;
    d.NN = 1 + c.pool + (c.depth - 1) * c.n_expand * c.pool;
    d.E = 1 + (c.depth - 1) * c.n_expand;
    if (16 * (size_t)(d.NN - 1) > 64 * 1024) {
        return fail(RHEO_EINVAL, "tree too large (%d nodes per sequence)", d.NN);
    }
    // expand variant: 16 vectors per thread and chunk (dense mode: 8, whose
    // twice as many chunk blocks run its selection and weight passes about
    // 4 % faster at the headline shape) unless the chunk lists would not fit
    // the merge; RHEO_EXPAND_VARIANT picks another that fits
    t->variant = -1;
    for (int v = dense ? 1 : 2; v < expand_variant_count(c.dtype); ++v) {
        if (variant_fits(c.dtype, v, c.vocab, SL, dense)) {
            t->variant = v;
            break;
        }
    }
    if (t->variant < 0) {
        return fail(RHEO_EINVAL, "vocab %d with support %d exceeds the expand merge capacity",
                    c.vocab, SL);
    }
    // sparse levels run one block per row (the row streamed once, no chunk
    // lists) when the row fits it and the level has at least row_min rows;
    // RHEO_EXPAND_ROW=0 or 1 forces the chunked or the per-row kernel
    t->row_mode = (!dense && expand_row_nq(c.dtype, c.vocab) > 0) ? -1 : 0;
    if (const char* er = getenv("RHEO_EXPAND_ROW")) {
        if (er[0] == '0') t->row_mode = 0;
        else if (er[0] == '1' && t->row_mode != 0) t->row_mode = 1;
    }
    if (const char* rm = getenv("RHEO_ROW_MIN")) t->row_min = atoi(rm);
    // levels with more rows than the device holds 512-thread row blocks at
    // once run 256-thread blocks (twice the vectors per thread, twice the
    // blocks resident); RHEO_ROW_NARROW=0 or 1 forces the choice
    t->dev.row_narrow = -1;
    if (const char* rn = getenv("RHEO_ROW_NARROW")) t->dev.row_narrow = rn[0] == '1' ? 1 : 0;
    const char* env = getenv("RHEO_EXPAND_VARIANT");
    if (env) {
        const int v = atoi(env);
        if (v >= 0 && v < expand_variant_count(c.dtype) &&
            variant_fits(c.dtype, v, c.vocab, SL, dense))
            t->variant = v;
    }
    {
        const ExpandVariant ev = expand_variant(c.dtype, t->variant, c.vocab, SL);
        d.C = ev.C;
        d.Sc = ev.Sc;
        if (d.Sc != SL) {   // chunks hold at least 4096 elements, lists at most 1024
                return fail(RHEO_EINVAL, "internal: expand chunk smaller than the support");
        }
    }
    return RHEO_OK;
}

// Where a tree's device arrays come from: device allocations (rheo_create),
// a region of the static scratch array (rheo_create_static), or nowhere
// (a measuring pass that only counts the bytes of the region).
struct Arena {
    enum Mode { HEAP, REGION, MEASURE } mode;
    rheo_tree* t;
    char* base = nullptr;        // REGION: start of the region
    size_t cap = 0, used = 0;    // REGION / MEASURE: bytes
    int rc = RHEO_OK;
};

template <typename T>
void take(Arena& A, T** p, size_t count) {
    if (A.rc) return;
    const size_t bytes = count * sizeof(T) ? count * sizeof(T) : 16;
    if (A.mode == Arena::HEAP) {
        A.rc = dalloc(A.t, p, count);
        return;
    }
    const size_t off = (A.used + 255) & ~(size_t)255;
    A.used = off + bytes;
    if (A.mode == Arena::MEASURE) return;
    if (A.used > A.cap) {
        A.rc = fail(RHEO_EINVAL, "internal: static region overrun");
        return;
    }
    *p = (T*)(A.base + off);
}

// Every device array of the tree, in one fixed order.
void layout(rheo_tree* t, Arena& A) {
    TreeDev& d = t->dev;
    const bool dense = d.dense != 0;
    const size_t B = d.B, NN = d.NN, E = d.E;
    take(A, &d.tok, B * NN);
    take(A, &d.par, B * NN);
    take(A, &d.meta, B * NN);
    take(A, &d.proxy, B * NN);
    take(A, &d.qtrue, B * NN);
    take(A, &d.score, B * NN);
    take(A, &d.path, B * NN);
    take(A, &d.first_child, B * NN);
    take(A, &d.exp_of, B * NN);
    take(A, &d.tidx, B * NN);
    const size_t TS = dense ? 1 : (size_t)d.S;              // dense mode keeps no tail copy
    take(A, &d.tail_id, B * E * TS);
    take(A, &d.tail_q, B * E * TS);
    const size_t DN = dense ? 1 : 0;
    take(A, &d.dq, DN ? B * d.NE * (size_t)d.NCH : 1);
    take(A, &d.dpart, DN ? B * d.NE * (size_t)d.C * 2 : 1);
    take(A, &d.dflag, DN ? B * d.NE : 1);
    take(A, &d.dref, DN ? B * E : 1);
    take(A, &d.dleads, DN ? B * E * 16 : 1);
    take(A, &d.zq, B * E);
    take(A, &d.s1row, d.cfull ? B * d.NE : 1);
    take(A, &d.frontier, B * d.NE);
    take(A, &d.fr_parent, B * d.NE);
    take(A, &d.fr_token, B * d.NE);
    take(A, &d.pidx, B * NN);
    take(A, &d.porder, B * NN);
    take(A, &d.err, 1);
    take(A, &d.team_ticket, B);
    take(A, &d.team_flag, B * 64);
    take(A, &d.team_max, B * 64);
    take(A, &d.team_sum, B * 64);
    take(A, &d.team_chunk, B * 1024);
    take(A, &d.team_sp, B * (1024 + 16));
    take(A, &d.team_nchunk, dense ? B * 1024 * 2 : 1);
    take(A, &d.sel, B * d.NE * (size_t)d.C * d.Sc);
    take(A, &d.seq_cnt, B);
}

// Clears what the kernels expect zeroed (or -1) before a tree's first step
// and picks the verification team shape.
int init_state(rheo_tree* t) {
    TreeDev& d = t->dev;
    const size_t B = d.B, NN = d.NN;
    const bool dense = d.dense != 0;
    hipError_t e = hipMemset(d.err, 0, sizeof(int32_t));
    if (e == hipSuccess) e = hipMemset(d.team_ticket, 0, B * sizeof(uint64_t));
    if (e == hipSuccess) e = hipMemset(d.team_flag, 0, B * 64 * sizeof(uint64_t));
    if (e == hipSuccess) e = hipMemset(d.team_max, 0, B * 64 * sizeof(uint64_t));
    if (e == hipSuccess) e = hipMemset(d.team_sum, 0, B * 64 * sizeof(uint64_t));
    if (e == hipSuccess) e = hipMemset(d.seq_cnt, 0, B * sizeof(uint32_t));
    if (e == hipSuccess && dense) e = hipMemset(d.dflag, 0, B * d.NE * sizeof(int32_t));
    if (e == hipSuccess) e = hipMemset(d.pidx, 0xFF, B * NN * sizeof(int32_t));
    if (e == hipSuccess) e = hipMemset(d.frontier, 0, B * d.NE * sizeof(int32_t));
    if (e == hipSuccess) e = hipMemset(d.first_child, 0xFF, B * NN * sizeof(int32_t));
    if (e == hipSuccess) e = hipDeviceSynchronize();
    if (e != hipSuccess) return hip_fail(e, "initialising tree state");
    e = verify_shape(d, &t->vG, &t->v_segch, &t->v_grid);
    if (e != hipSuccess) return hip_fail(e, "no co-resident verification team shape for this tree");
    e = expand_row_slots(d, &d.row_slots);
    if (e != hipSuccess) return hip_fail(e, "row kernel occupancy");
    return RHEO_OK;
}

// ---------------------------------------------------------------------------
// The static scratch array of rheo_create_static: a tree's whole device state
// without any allocation.  Each device that loads the library holds its own
// copy until the process ends.  Host code never passes the array's name to
// a kernel or copy (on the host it is only a stand-in for the symbol): the
// device address comes from hipGetSymbolAddress, taken once per device with
// that device current.
// ---------------------------------------------------------------------------
constexpr size_t kScratchBytes = (size_t)32 << 20;
constexpr int kMaxDevices = 64;

}  // namespace

static __device__ __align__(256) char scratch[kScratchBytes];

namespace {

char* g_region[kMaxDevices];              // device address of `scratch`, per device
std::mutex g_region_mu;
rheo_tree g_static[kMaxDevices];          // the static handle of each device

int static_region(int dev, char** region) {
    std::lock_guard<std::mutex> lock(g_region_mu);
    if (!g_region[dev]) {
        void* ptr = nullptr;
        const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
        if (!ptr) return fail(RHEO_EHIP, "hipGetSymbolAddress(scratch) returned NULL");
        g_region[dev] = (char*)ptr;
    }
    *region = g_region[dev];
    return RHEO_OK;
}

}  // namespace

extern "C" {

const char* rheo_last_error(void) { return g_err.c_str(); }

int rheo_create(const rheo_config* cfg, rheo_tree** out) {
    if (!cfg || !out) return fail(RHEO_EINVAL, "NULL argument");
    rheo_tree* t = new rheo_tree();
    int rc = configure(cfg, t);
    if (rc == RHEO_OK) {
        Arena A{Arena::HEAP, t};
        layout(t, A);
        rc = A.rc;
    }
    if (rc == RHEO_OK) rc = init_state(t);
    if (rc != RHEO_OK) {
        free_all(t);
        delete t;
        return rc;
    }
    *out = t;
    return RHEO_OK;
}

int rheo_create_static(const rheo_config* cfg, rheo_tree** out) {
    if (!cfg || !out) return fail(RHEO_EINVAL, "NULL argument");
    // validate and measure on a staging copy first, so that a refused call
    // makes no device call and leaves the device's static handle as it was
    rheo_tree stage;
    int rc = configure(cfg, &stage);
    if (rc) return rc;
    Arena M{Arena::MEASURE, &stage};
    layout(&stage, M);
    if (M.used > kScratchBytes)
        return fail(RHEO_EINVAL, "tree needs %zu bytes of device state; the static scratch "
                    "holds %zu", M.used, (size_t)kScratchBytes);
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices) return fail(RHEO_EINVAL, "device %d out of range", dev);
    char* region = nullptr;
    rc = static_region(dev, &region);
    if (rc) return rc;
    rheo_tree& t = g_static[dev];
    t = stage;
    t.is_static = true;
    Arena A{Arena::REGION, &t, region, (size_t)kScratchBytes};
    layout(&t, A);
    if (A.rc) return A.rc;
    rc = init_state(&t);
    if (rc) return rc;
    *out = &t;
    return RHEO_OK;
}

int rheo_destroy(rheo_tree* t) {
    if (!t) return RHEO_OK;
    (void)hipDeviceSynchronize();
    if (t->is_static) return RHEO_OK;      // the static scratch stays with the device
    free_all(t);
    delete t;
    return RHEO_OK;
}

int32_t rheo_node_count(const rheo_tree* t) { return t ? t->dev.NN : 0; }

int rheo_begin_step(rheo_tree* t) {
    if (!t) return fail(RHEO_EINVAL, "NULL tree");
    t->state = EXPANDING;
    t->level = 0;
    t->R = 0;
    return RHEO_OK;
}

int rheo_expand_level(rheo_tree* t, const void* logits, float T, uint64_t key, void* stream) {
    if (!t) return fail(RHEO_EINVAL, "NULL tree");
    if (t->state != EXPANDING) return fail(RHEO_ESTATE, "rheo_expand_level needs rheo_begin_step first");
    int rc = check_ptr(logits, "draft_logits");
    if (rc) return rc;
    if ((rc = check_T(T))) return rc;
    if (t->level == 0) {
        t->T_step = T;
        t->key_step = key;
    } else if ((rc = check_step_args(t, T, key, "rheo_expand_level"))) {
        return rc;
    }
    LevelArgs a;
    a.logits = logits;
    a.level = t->level;
    a.P = t->level == 0 ? 1 : t->dev.NE;
    a.k1 = k_of_T(t->cfg.construct_tempered ? T : 1.0f);
    a.kT = k_of_T(T);
    a.rng_key = key;
    a.fr_key = key;                       // the key of the call that chose the parents
    hipError_t e = hipSuccess;
    if (t->dev.cfull) {
        // the construction totals over the whole rows, read by the pools
        e = launch_row_wsum(t->dev, a, (hipStream_t)stream);
        if (e != hipSuccess) return hip_fail(e, "row total launch");
    }
    if (t->dev.dense) {
        e = launch_select(t->dev, a, t->variant, (hipStream_t)stream);
        if (e == hipSuccess)
            e = launch_dense(t->dev, a, expand_variant_nvc(t->variant), (hipStream_t)stream);
    } else if (t->row_mode == 1 || (t->row_mode < 0 && t->dev.B * a.P >= t->row_min)) {
        e = launch_expand_row(t->dev, a, (hipStream_t)stream);
    } else {
        e = launch_expand(t->dev, a, t->variant, (hipStream_t)stream);
    }
    if (e != hipSuccess) return hip_fail(e, "expand launch");
    t->draft[t->level] = logits;
    if (++t->level == t->dev.D) t->state = EXPANDED;
    return RHEO_OK;
}

int rheo_frontier(rheo_tree* t, int32_t* parent_index, int32_t* token, void* stream) {
    if (!t) return fail(RHEO_EINVAL, "NULL tree");
    if (t->state != EXPANDING || t->level < 1)
        return fail(RHEO_ESTATE, "no frontier: expand a level below the last first");
    const size_t bytes = (size_t)t->dev.B * t->dev.NE * sizeof(int32_t);
    hipError_t e = hipSuccess;
    if (parent_index)
        e = hipMemcpyAsync(parent_index, t->dev.fr_parent, bytes, hipMemcpyDeviceToDevice,
                           (hipStream_t)stream);
    if (e == hipSuccess && token)
        e = hipMemcpyAsync(token, t->dev.fr_token, bytes, hipMemcpyDeviceToDevice,
                           (hipStream_t)stream);
    return e == hipSuccess ? RHEO_OK : hip_fail(e, "frontier copy");
}

int rheo_frontier_view(const rheo_tree* t, const int32_t** parent_index, const int32_t** token) {
    if (!t || !parent_index || !token) return fail(RHEO_EINVAL, "NULL argument");
    *parent_index = t->dev.fr_parent;
    *token = t->dev.fr_token;
    return RHEO_OK;
}

int rheo_prune(rheo_tree* t, int32_t R, void* stream) {
    if (!t) return fail(RHEO_EINVAL, "NULL tree");
    if (t->state != EXPANDED) return fail(RHEO_ESTATE, "rheo_prune needs all depth levels expanded");
    if (R < 1 || R > t->dev.NN - 1) return fail(RHEO_EINVAL, "budget must be in [1, %d]", t->dev.NN - 1);
    const hipError_t e = launch_prune(t->dev, R, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "prune launch");
    t->R = R;
    t->state = PRUNED;
    return RHEO_OK;
}

int rheo_pruned_view(rheo_tree* t, int32_t* parent, int32_t* token, void* stream) {
    if (!t) return fail(RHEO_EINVAL, "NULL tree");
    if (t->state != PRUNED && t->state != VERIFIED) return fail(RHEO_ESTATE, "no pruned tree");
    const hipError_t e = launch_pruned_view(t->dev, t->R, parent, token, (hipStream_t)stream);
    return e == hipSuccess ? RHEO_OK : hip_fail(e, "pruned view launch");
}

int rheo_tree_mask(rheo_tree* t, uint8_t* mask, int32_t* depth, void* stream) {
    if (!t) return fail(RHEO_EINVAL, "NULL tree");
    if (t->state != PRUNED && t->state != VERIFIED) return fail(RHEO_ESTATE, "no pruned tree");
    const hipError_t e = launch_tree_mask(t->dev, t->R, mask, depth, (hipStream_t)stream);
    return e == hipSuccess ? RHEO_OK : hip_fail(e, "tree mask launch");
}

int rheo_verify(rheo_tree* t, const void* logits, float T, uint64_t key, int32_t* accepted,
                int32_t* accept_len, int32_t* final_token, void* stream) {
    if (!t) return fail(RHEO_EINVAL, "NULL tree");
    if (t->state != PRUNED) return fail(RHEO_ESTATE, "rheo_verify needs rheo_prune first");
    int rc = check_ptr(logits, "target_logits");
    if (rc) return rc;
    if ((rc = check_T(T))) return rc;
    if ((rc = check_step_args(t, T, key, "rheo_verify"))) return rc;
    if (!accepted || !accept_len || !final_token) return fail(RHEO_EINVAL, "NULL output");
    VerifyArgs a;
    a.logits = logits;
    a.R = t->R;
    a.kT = k_of_T(T);
    a.rng_key = key;
    a.accepted = accepted;
    a.accept_len = accept_len;
    a.final_token = final_token;
    a.G = t->vG;
    for (int i = 0; i < 16; ++i) a.draft[i] = t->draft[i];
    // about a second of polling; RHEO_VERIFY_SPIN (read at each call) lowers
    // it, so that tests can force the failure path from the host
    a.spin = 1L << 20;
    if (const char* sp = getenv("RHEO_VERIFY_SPIN")) a.spin = atol(sp);
    const hipError_t e = launch_verify(t->dev, a, t->v_segch, t->v_grid, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "verify launch");
    t->state = VERIFIED;
    return RHEO_OK;
}

int rheo_read_nodes(rheo_tree* t, int32_t* token, int32_t* parent, int32_t* depth, int32_t* slot,
                    int32_t* kind, double* proxy, double* qtrue, double* score, void* stream) {
    if (!t) return fail(RHEO_EINVAL, "NULL tree");
    if (t->state == CREATED || (t->state == EXPANDING && t->level == 0))
        return fail(RHEO_ESTATE, "no tree built in this step");
    const hipError_t e = launch_read_nodes(t->dev, token, parent, depth, slot, kind, proxy, qtrue,
                                           score, (hipStream_t)stream);
    return e == hipSuccess ? RHEO_OK : hip_fail(e, "read_nodes launch");
}

int rheo_device_error(rheo_tree* t, int32_t* host_flag) {
    if (!t || !host_flag) return fail(RHEO_EINVAL, "NULL argument");
    hipError_t e = hipDeviceSynchronize();
    if (e == hipSuccess) e = hipMemcpy(host_flag, t->dev.err, sizeof(int32_t), hipMemcpyDeviceToHost);
    return e == hipSuccess ? RHEO_OK : hip_fail(e, "reading the device error flag");
}

}  // extern "C"
