/*
 * rheo.h -- C ABI of the RheoSampling hot path on AMD Instinct MI355X (gfx950).
 *
 * RheoSampling (arXiv 2609.21827) builds a speculative-decoding draft tree by
 * EAGLE's expand-then-rerank (Sec. 2.1) with one stochastic slot per candidate
 * pool: the top-m draft tokens, then one token Y sampled from the tail
 * distribution q~, then the highest-ranked remaining tokens (Sec. 3.2, "Hybrid
 * sampling mechanism"; App. C.1).  Y competes in expansion and pruning with
 * the proxy probability min{q(x_m), z} and is verified with its true
 * probability q~(Y) (Sec. 3.2, "Dual treatment").  The tree is pruned globally
 * to R nodes by path score with a fixed tie-break (App. C.1) and verified
 * layer by layer by RheoVerification (Algorithm 1; Thm. 1).
 *
 * One decoding step for B independent sequences is
 *     rheo_begin_step
 *     rheo_expand_level  x depth     (draft logits of the current frontier)
 *     rheo_prune
 *     rheo_verify                    (target logits of the pruned tree)
 * and the caller runs its draft / target model between the calls, using
 * rheo_frontier and rheo_pruned_view to learn which rows to compute.
 *
 * Conventions
 *   - All data pointers are device pointers (HBM) unless marked "host".
 *     The caller owns every logit and output buffer; the tree handle owns its
 *     own device state, sized at rheo_create.
 *   - Every call that takes a stream enqueues work on that HIP stream
 *     (hipStream_t, passed as void*; NULL = the default stream) and returns
 *     without synchronising.  A handle must not be used from two streams at
 *     once; calls on one handle must follow the step order above.
 *   - Return value: RHEO_OK or a negative error code; rheo_last_error()
 *     gives a message for the calling thread's last failure.  Arguments are
 *     validated on the host before anything is enqueued, so an error leaves
 *     the device state as it was.
 *   - Logit rows: dtype RHEO_F32 or RHEO_BF16, V contiguous elements per row,
 *     consecutive rows row_stride elements apart, base pointer 16-byte aligned
 *     and row_stride a multiple of 16 bytes.  A logit is finite or -inf (a
 *     masked token, the truncation of Sec. 3.2: probability 0).  NaN and
 *     +inf are not allowed and not checked.  Device error bit 9 (512)
 *     reports the cases where the method is undefined: a draft row whose
 *     x_{m+1} (the (m+1)-th token by construction weight, ties by id) has
 *     logit -inf, so q~_T has no reference; a target row with no finite
 *     logit (see rheo_verify).
 *   - Decisions are exact: each probability is an integer weight (a
 *     fixed-point softmax numerator evaluated by a fixed fp32 operation
 *     sequence), sums are exact 64-bit integers and every sampling or
 *     acceptance decision is an exact integer comparison, so results do not
 *     depend on launch shapes or reduction order.  Random draws are
 *     Philox4x64-10 (Salmon et al., SC'11) blocks keyed by rng_key with the
 *     counter (index, sequence, purpose, 0), purposes 1 = the sampled token
 *     of the node with uid index, 2 = acceptance test 32*level + j (j = 0 for
 *     the sampled child, else the candidate's slot), 3 = the final sample of
 *     a level.
 */
#ifndef RHEO_H
#define RHEO_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct rheo_tree rheo_tree;

enum {
    RHEO_OK = 0,
    RHEO_EINVAL = -1,   /* invalid argument or configuration             */
    RHEO_ENOMEM = -2,   /* device allocation failed                      */
    RHEO_EHIP = -3,     /* a HIP runtime call failed (message attached)  */
    RHEO_ESTATE = -4    /* call out of the step order                    */
};

enum { RHEO_F32 = 0, RHEO_BF16 = 1 };

enum { RHEO_METHOD_RHEO = 0, RHEO_METHOD_RRSW = 1, RHEO_METHOD_TOPK = 2 };

typedef struct rheo_config {
    int32_t batch;               /* B >= 1 independent sequences                      */
    int32_t vocab;               /* V, 2 <= V <= 262143                               */
    int32_t pool;                /* K slots per candidate pool, sampled slot included
                                    (Sec. 3.2); 1 <= K <= 15                           */
    int32_t leads;               /* m deterministic lead tokens, 0 <= m <= K-1          */
    int32_t depth;               /* D expansion levels, 1 <= D <= 15                   */
    int32_t n_expand;            /* parents expanded per level below the root,
                                    1..K (EAGLE expands K, Sec. 2.1); 0 means K         */
    int32_t support;             /* S: draft logits truncated to their top-S entries
                                    before the softmax (Sec. 3.2, sparse draft; the
                                    paper uses 128, App. B).  K <= S <= 1024.
                                    S <= 0 selects dense mode: the support is the whole
                                    vocabulary, and verification re-reads the draft
                                    rows (see rheo_expand_level)                        */
    int32_t construct_tempered;  /* 0: tree built on untempered q (Sec. 5.4);
                                    1: on the tempered q_T                              */
    int32_t dtype;               /* RHEO_F32 or RHEO_BF16                               */
    int32_t method;              /* RHEO_METHOD_RHEO: the pools of Sec. 3.2 verified by
                                    Algorithm 1 (the sampled child first);
                                    RHEO_METHOD_RRSW: the same pools verified leads
                                    first -- the leads under p, then the sampled child
                                    under what remains, then the fills under
                                    norm(max(0, r - q~)) (App. D.2);
                                    RHEO_METHOD_TOPK: pure top-K pools, no sampled
                                    slot (Sec. 2.1), sequential tests under p        */
    int32_t construct_full;      /* sparse mode: 0 builds the tree on q truncated to
                                    the support (Sec. 3.2); 1 on q over the whole
                                    vocabulary, the support then limiting only the
                                    sampled token's tail q~ and verification (the
                                    reading of Sec. 5.5 that truncation touches only
                                    the sampled token).  Costs one extra read of each
                                    draft row.  0 or 1; no effect in dense mode     */
    int64_t row_stride;          /* elements between consecutive logit rows (>= V)     */
    double eps_m0;               /* epsilon of the m = 0 proxy q(x_1) + eps (Sec. 3.2);
                                    0 selects 2^-40                                     */
} rheo_config;

/* Allocates a tree for cfg (host pointer, copied).  *out receives the handle.
 * Node capacity per sequence: 1 + K + (D-1) * n_expand * K.
 * Launch shapes, read from the environment here and never changing a
 * result: RHEO_EXPAND_ROW (0: sparse levels on the chunked kernel pair, 1:
 * on the one-block-per-row kernel wherever the row fits it), RHEO_ROW_MIN
 * (fewest rows of a level for the per-row kernel, default 1),
 * RHEO_ROW_NARROW (1 or 0: the per-row kernel's 256-thread blocks always or
 * never; by default when a level has more rows than the device holds
 * 512-thread blocks at once), RHEO_EXPAND_VARIANT (chunk size of the
 * chunked pair), RHEO_VERIFY_BLOCKS (blocks of all verification teams,
 * default 1024, capped by what the device holds at once).  RHEO_VERIFY_SPIN,
 * read at each rheo_verify, sets the polls of a team wait before it gives up
 * (see rheo_verify). */
int rheo_create(const rheo_config* cfg, rheo_tree** out);

/* rheo_create for callers that cannot allocate device memory (serving loops
 * and harnesses that forbid hipMalloc): the tree's whole device state lives
 * in a static array of the library, 32 MiB per device, which every device
 * that loads the library holds until the process ends.  No device memory is
 * allocated or freed.  A configuration whose state exceeds 32 MiB returns
 * RHEO_EINVAL before any device call (the five workload shapes of the
 * sparse and dense modes fit; supports of 512 and more at large batches do
 * not).  There is one static tree per device (the current device): every
 * call on a device re-initialises it and returns the same handle in *out, so
 * a static tree from an earlier call on that device becomes this one.
 * Calls on one device that overlap -- two threads creating, or work still
 * using the earlier static tree -- race.  The call synchronises the device
 * (not for use under graph capture); the handle's other calls behave as for
 * rheo_create, and rheo_destroy on it only synchronises. */
int rheo_create_static(const rheo_config* cfg, rheo_tree** out);

/* Frees the handle and its device memory (synchronises the device); for the
 * handle of rheo_create_static it frees nothing. */
int rheo_destroy(rheo_tree* tree);

/* Starts a new step: the next rheo_expand_level builds level 0 from the root. */
int rheo_begin_step(rheo_tree* tree);

/* Expands the current frontier by one level (Sec. 2.1 with the pools of
 * Sec. 3.2 / App. C.1).
 *   draft_logits  [B][P][row_stride] of cfg.dtype, P = 1 at level 0 (the
 *                 root) and n_expand afterwards; row (b, j) holds the draft
 *                 model's logits at frontier node j of sequence b.
 *   T             sampling temperature (> 0, finite): Y ~ q~_T.
 *   rng_key       key of the step's Philox draws.
 * T and rng_key are fixed for the whole step: the first call of a step sets
 * them, and a later rheo_expand_level or the step's rheo_verify with another
 * value returns RHEO_EINVAL (the stored tail weights and the draws of the
 * sampled slots depend on both).
 * Writes K children per frontier node (token, proxy, true probability,
 * path score) and, below the last level, selects the n_expand children with
 * the highest path scores as the next frontier.  With support S, the
 * truncated distribution is kept in the tree for verification, so the
 * draft buffer may be reused as soon as this call's work has run.  In dense
 * mode the tree borrows draft_logits: verification re-reads the rows of the
 * nodes it walks, so the buffer of every level must stay allocated and
 * unchanged until the step's rheo_verify has run on its stream. */
int rheo_expand_level(rheo_tree* tree, const void* draft_logits, float T,
                      uint64_t rng_key, void* stream);

/* The frontier chosen by the last rheo_expand_level, in rank order, copied
 * into caller buffers on `stream`:
 *   parent_index  [B][n_expand] int32: index of the node's parent in the
 *                 previous frontier (0 at level 1)
 *   token         [B][n_expand] int32: the node's token
 * (device pointers; either may be NULL).  Valid below the last level.
 * RHEO_ESTATE if no level below the last has been expanded in this step. */
int rheo_frontier(rheo_tree* tree, int32_t* parent_index, int32_t* token,
                  void* stream);

/* The same frontier without a copy: *parent_index and *token receive the
 * tree-owned device arrays ([B][n_expand] int32 each, layout as above).  The
 * pointers stay fixed for the life of the handle; their contents are those
 * of the last rheo_expand_level below the last level, once that call's
 * work has run on its stream, until the next such call.  Host-only: no
 * device work, no synchronisation. */
int rheo_frontier_view(const rheo_tree* tree, const int32_t** parent_index,
                       const int32_t** token);

/* Keeps the budget R best non-root nodes (1 <= R <= K + (D-1) n_expand K) by
 * path score, ties by depth (shallower first) then left-to-right sibling
 * order (App. C.1); the root does not count towards R. */
int rheo_prune(rheo_tree* tree, int32_t budget, void* stream);

/* The pruned tree in rank order, index 0 = root:
 *   parent  [B][R+1] int32 (pruned index of the parent, -1 for the root)
 *   token   [B][R+1] int32 (-1 for the root)
 * Row i of the target buffer given to rheo_verify must hold the target
 * model's logits at pruned node i. */
int rheo_pruned_view(rheo_tree* tree, int32_t* parent, int32_t* token,
                     void* stream);

/* What the target model needs to score the pruned tree in one forward
 * pass, all drafted paths at once (Sec. 1; Sec. 2.1), in pruned order.
 * Valid after rheo_prune.  Either pointer may be NULL.
 *   mask   [B][R+1][R+1] uint8: mask[b][i][j] = 1 iff pruned node j is on
 *          the path from the root to pruned node i (i included), else 0.
 *          Parents precede their children in pruned order, so the mask is
 *          lower triangular.
 *   depth  [B][R+1] int32: depth of each pruned node (root 0), its
 *          position after the prefix.
 * Buffers are the caller's, written completely. */
int rheo_tree_mask(rheo_tree* tree, uint8_t* mask, int32_t* depth, void* stream);

/* RheoVerification (Algorithm 1) applied layer by layer from the root
 * (Thm. 1), with p = softmax(target / T) over the whole vocabulary.
 *   target_logits [B][R+1][row_stride] of cfg.dtype (pruned-node order)
 *   accepted      [B][depth] int32: accepted draft tokens, -1 after the end
 *   accept_len    [B] int32: number of accepted draft tokens
 *   final_token   [B] int32: the token emitted after them (residual sample,
 *                 or a sample of p below an accepted leaf)
 * The output of a step is accepted[0..accept_len) followed by final_token.
 * T and rng_key must be the step's (see rheo_expand_level), else RHEO_EINVAL.
 * The kernel's blocks wait for each other (teams of blocks per sequence);
 * its grid never exceeds what the device holds at once, so on a device that
 * runs nothing else at the same time every wait completes.  Work running
 * concurrently on the same device can delay some blocks: a wait longer than
 * about a second then ends that sequence's walk with the failure result
 * accept_len[b] = final_token[b] = -1 and accepted[b][*] = -1, and sets
 * device error bit 7 (128).  Callers check accept_len >= 0; a failed
 * sequence's step is not Algorithm 1's and must be run again.  A walk that
 * reaches a node whose target row has no finite logit (p undefined) ends
 * with the same failure result and sets device error bit 9 (512). */
int rheo_verify(rheo_tree* tree, const void* target_logits, float T,
                uint64_t rng_key, int32_t* accepted, int32_t* accept_len,
                int32_t* final_token, void* stream);

/* Copies the unpruned tree of the current step (uid order, [B][N], N =
 * 1 + K + (D-1) n_expand K, uid 0 = root; children of a level are numbered
 * in frontier order, then slot order).  Any pointer may be NULL.
 *   kind: 0 lead, 1 sampled, 2 fill; qtrue: q~(Y) for the sampled slot,
 *   q(x) for the others; score: product of proxies from the root. */
int rheo_read_nodes(rheo_tree* tree, int32_t* token, int32_t* parent,
                    int32_t* depth, int32_t* slot, int32_t* kind,
                    double* proxy, double* qtrue, double* score, void* stream);

/* Synchronises the device and copies the tree's sticky device error flag to
 * *host_flag (0 = no error; bit 0: no sampled token found, bit 1: pruned
 * tree not ancestor-closed, bit 2: sampled child missing from its parent's
 * tail, bit 3: residual sample out of range, bit 4: corrupt frontier,
 * bit 5: corrupt verification walk, bit 6: invalid launch shape, bit 7:
 * verification team barrier timed out, bit 8: a support slot left empty by
 * the expand merge, bit 9: a draft row whose x_{m+1} is -inf or a target
 * row without a finite logit).
 * Diagnostic only. */
int rheo_device_error(rheo_tree* tree, int32_t* host_flag);

/* Nodes per sequence of the unpruned tree (root included). */
int32_t rheo_node_count(const rheo_tree* tree);

/* Message of the calling thread's last failed call ("" if none). */
const char* rheo_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* RHEO_H */
