// Device state of one tree handle and the kernel launch entry points.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rheo {

// Everything a kernel needs to find the tree arrays.  Node arrays are
// [B][NN] in uid order (uid 0 = root); expanded-node arrays are [B][E] with
// expanded index e = 0 for the root and 1 + (d-1) * NE + j for frontier
// node j of level d >= 1.
struct TreeDev {
    int B, V, K, m, D, NE, S;      // S = effective support (min(S, V))
    int NN, E;                      // nodes / expanded nodes per sequence
    int dtype;
    int64_t stride;
    double eps;
    // unpruned tree, [B][NN]
    int32_t* tok;
    int32_t* par;
    int32_t* meta;                 // depth | slot << 8 | kind << 16
    double* proxy;
    double* qtrue;
    double* score;
    uint64_t* path;                // slot path, 4 bits per level from bit 59 down
    int32_t* first_child;          // uid of slot-1 child, -1 if not expanded
    int32_t* exp_of;               // expanded index, -1 if not expanded
    int32_t* tidx;                 // place in the parent's stored tail (sparse), else -1
    // truncated tail distribution q~ of each expanded node, sorted by id
    int32_t* tail_id;              // [B][E][S]
    uint32_t* tail_q;              // [B][E][S]
    uint64_t* zq;                  // [B][E]
    // frontier of the last expanded level, [B][NE]: node uid, index of its
    // parent in the previous frontier, token
    int32_t* frontier;
    int32_t* fr_parent;
    int32_t* fr_token;
    // pruned tree
    int32_t* pidx;                 // [B][NN]: pruned index, -1 if pruned away
    int32_t* porder;               // [B][NN]: uid of each pruned index
    int32_t* err;                  // sticky device error flag
    // verification team exchange (see verify.hip)
    uint64_t* team_ticket;         // [B] blocks of each team so far (monotonic)
    uint64_t* team_flag;           // [B][GMAX] arrival epochs
    uint64_t* team_max;            // [B][GMAX] segment maxima: epoch << 32 | order code
    uint64_t* team_sum;            // [B][GMAX] segment weight sums: epoch << 48 | sum
    uint64_t* team_chunk;          // [B][NCMAX] chunk totals of p's weights
    uint32_t* team_sp;             // [B][SPMAX] p's weights at the special tokens
    uint64_t* team_nchunk;         // dense: [B][NCMAX][2] residual chunk totals (u128)
    // expansion: each row's C chunk lists of Sc selection keys, sorted
    uint64_t* sel;                 // [B * NE][C][Sc]
    // dense mode (the support is all of V): per row the tail-weight totals
    // of each 64-vector sub-chunk, the chunks' sums (w1, q) and the rank-tie
    // flag; per expanded node the logit of x_{m+1} and the leads
    int dense;
    int NCH;                       // sub-chunks per row (dense)
    uint64_t* dq;                  // [B * NE][NCH]
    uint64_t* dpart;               // [B * NE][C][2]
    int32_t* dflag;                // [B * NE]
    float* dref;                   // [B][E]
    int32_t* dleads;               // [B][E][16]
    uint32_t* seq_cnt;             // [B] rows whose pool is written (0 between launches)
    int C, Sc;
    int rrsw;                      // verification leads first (App. D.2)
    int topk;                      // pure top-K pools, no sampled slot
    int cfull;                     // construction over the whole vocabulary (sparse)
    int row_slots;                 // 512-thread row-kernel blocks the device holds at once
    int row_narrow;                // 256-thread row blocks: 1 always, 0 never, -1 above row_slots
    uint64_t* s1row;               // [B * NE]: its total per row of the level
};

struct LevelArgs {
    const void* logits;
    int level;                     // 0..D-1
    int P;                         // parents per sequence at this level
    float k1;                      // construction kT (untempered unless asked)
    float kT;                      // sampling kT
    uint64_t rng_key;
    uint64_t fr_key;               // rng_key of the launch that chose this level's parents
};

struct VerifyArgs {
    const void* logits;
    const void* draft[16];         // dense: each level's draft rows (borrowed)
    int R;
    int G;                         // blocks per sequence (a team)
    int NV;                        // chunks per segment
    float kT;
    uint64_t rng_key;
    long spin;                     // polls of a team wait before it gives up
    int32_t* accepted;
    int32_t* accept_len;
    int32_t* final_token;
};

hipError_t launch_expand(const TreeDev& t, const LevelArgs& a, int variant,
                         hipStream_t s);
hipError_t launch_select(const TreeDev& t, const LevelArgs& a, int variant, hipStream_t s);
hipError_t launch_dense(const TreeDev& t, const LevelArgs& a, int nvc, hipStream_t s);
hipError_t launch_prune(const TreeDev& t, int R, hipStream_t s);
hipError_t verify_shape(const TreeDev& t, int* G, int* segch, int* grid);
hipError_t launch_verify(const TreeDev& t, const VerifyArgs& a, int segch, int grid,
                         hipStream_t s);

// expand kernel variants: the chunk each selection block holds in registers
struct ExpandVariant {
    int chunk;                     // elements per chunk
    int C;                         // chunks per row
    int Sc;                        // selection keys kept per chunk
    bool ok;                       // the row's C * Sc keys fit the merge
};
hipError_t launch_expand_row(const TreeDev& t, const LevelArgs& a, hipStream_t s);
hipError_t launch_row_wsum(const TreeDev& t, const LevelArgs& a, hipStream_t s);
hipError_t launch_tree_mask(const TreeDev& t, int R, uint8_t* mask, int32_t* depth,
                            hipStream_t s);
int expand_row_nq(int dtype, int V);
hipError_t expand_row_slots(const TreeDev& t, int* slots);
int expand_variant_count(int dtype);
int expand_variant_nvc(int v);
ExpandVariant expand_variant(int dtype, int v, int V, int S);

}  // namespace rheo

namespace rheo {
hipError_t launch_read_nodes(const TreeDev& t, int32_t* token, int32_t* parent,
                             int32_t* depth, int32_t* slot, int32_t* kind, double* proxy,
                             double* qtrue, double* score, hipStream_t s);
hipError_t launch_pruned_view(const TreeDev& t, int R, int32_t* parent, int32_t* token,
                              hipStream_t s);
}  // namespace rheo
