/*
 * pctree.h -- C ABI of the PCTree per-round draft-tree builder for MI355X (gfx950).
 *
 * One speculative-decoding round of PCTree (Li et al., "From Chains to Trees:
 * Parent-Conditioned Drafting for Semi-Autoregressive Speculative Decoding")
 * turns shared backbone logits L_0..L_{B-1} into a budgeted draft tree:
 *
 *   for every depth d (Sec. 4.1, Alg. 1): the frontier parents are batched
 *   through the Markov head, z_d(p) = L_d + Markov(p) (Eq. 3), each row is
 *   log-softmax normalised (Eq. 2), every parent keeps its top-k children with
 *   joint path scores s(child) = s(p) + log pi_d(child|p) (Eq. 4), and the k
 *   best candidates of the layer become the next frontier; after B stages the
 *   global top-N of the pool (score desc, depth asc, stable id; Sec. 4.2) is
 *   emitted as flat tokens, parent indices, position ids and the ancestor-only
 *   tree attention mask (App. A).
 *
 * The Markov head is Markov_d(p) = W^T . SiLU(E[p] + h_d) with E[V][r],
 * W[r][V] and a per-depth feature h_d[r]; the paper gives only that the head
 * is low-rank and adds a bias set by the preceding token (Sec. 3.2).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Every data pointer is a DEVICE pointer on the current HIP device; the
 *    caller owns all memory, the library never allocates or frees.  Inputs
 *    are never written.  Outputs must not overlap inputs or the workspace.
 *  - Data pointers must be 16-byte aligned; the workspace 256-byte aligned.
 *  - `stream` is a hipStream_t (NULL = the default stream).  Calls only
 *    enqueue work: they return before the GPU has run it, do no host<->device
 *    copies and never synchronise.  Results are valid once the stream reaches
 *    that point.  Calls are re-entrant; concurrent calls need distinct
 *    workspaces.  Exception: a round with at most 16 frontier rows (R * k'
 *    <= 16) runs as ONE launch whose workgroups, one per compute unit,
 *    exchange data while they run, so they must all be resident together.
 *    Such rounds must not overlap another round (or other long kernels) on
 *    the same device, e.g. on a second stream: a workgroup that cannot start
 *    makes the others' bounded waits give up (after 2 s), and the round is
 *    then abandoned (see pctree_tree.count).  Rounds on one stream are
 *    always safe.
 *  - Argument checking happens on the host before anything is enqueued; on
 *    any error status no device work has been issued and nothing is written.
 *    No C++ exception crosses this interface.
 *  - Device-side data errors do not fault: a request whose root token lies
 *    outside [0, V) is emitted as an empty tree (count = 0, rows padded).
 *    Floating-point inputs must be finite.
 */
#ifndef PCTREE_H
#define PCTREE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define PCTREE_ABI_VERSION 1

/* Compiled limits (PCTREE_ERR_UNSUPPORTED beyond them). */
#define PCTREE_MAX_VOCAB (1 << 20)
#define PCTREE_MAX_BLOCK 63
#define PCTREE_MAX_TOPK 16
#define PCTREE_MAX_BUDGET 256
#define PCTREE_MAX_REQUESTS 256
#define PCTREE_MAX_RANK_BF16 512 /* and rank % 32 == 0 */
#define PCTREE_MAX_RANK_F32 128  /* and rank % 16 == 0 */
#define PCTREE_MAX_MASK_BUDGET 1024

typedef enum pctree_status {
  PCTREE_OK = 0,
  PCTREE_ERR_INVALID_ARGUMENT = 1, /* null pointer, size < 1, bad dtype, misaligned pointer */
  PCTREE_ERR_UNSUPPORTED = 2,      /* beyond the compiled limits, or an unknown mode */
  PCTREE_ERR_WORKSPACE = 3,        /* workspace null, too small or not 256-byte aligned */
  PCTREE_ERR_HIP = 4               /* a kernel launch failed */
} pctree_status;

typedef enum pctree_dtype {
  PCTREE_F32 = 0, /* float32 base logits and head weights */
  PCTREE_BF16 = 1 /* bfloat16 base logits and head weights, fp32 accumulation */
} pctree_dtype;

/* Scoring of a parent's children (Sec. 5.3 compares the three).  Other
 * values are PCTREE_ERR_UNSUPPORTED. */
typedef enum pctree_mode {
  PCTREE_MODE_PARENT = 0,      /* PCTree: every frontier parent p gets its own row
                                  z_d(p) = L_d + Markov_d(p) (Eq. 3)              */
  PCTREE_MODE_SHARED = 1,      /* Shared-Markov tree: the greedy chain of Eq. 1 is
                                  built first and its row at depth d,
                                  z_d(y_{d-1}), serves every parent of depth d     */
  PCTREE_MODE_INDEPENDENT = 2  /* parent-independent per-position scoring (the
                                  DDTree-style scoring named in Sec. 4): every parent
                                  of depth d gets log_softmax(L_d)               */
} pctree_mode;

/* Problem size of one round (symbols of Sec. 4.1). */
typedef struct pctree_shape {
  int32_t vocab;    /* V: vocabulary size                                    */
  int32_t block;    /* B: block size = number of sequential Markov stages    */
  int32_t budget;   /* N: verification node budget, root included            */
  int32_t topk;     /* k: local branching factor (k' = min(k, V) is used)    */
  int32_t rank;     /* r: Markov-head rank                                   */
  int32_t requests; /* R: independent requests built in one call             */
  int32_t dtype;    /* pctree_dtype of base_logits, emb and proj_t           */
  int32_t mode;     /* pctree_mode: how each parent's child row is scored      */
} pctree_shape;

/* Inputs of one round.  Request i uses base_logits[i], depth_feat[i],
 * root_token[i] and prefix_len[i]; emb and proj_t are one drafter's head,
 * shared by every request. */
typedef struct pctree_inputs {
  const void* base_logits;   /* L   [R][B][V] dtype: backbone logits L_d (Sec. 3.2)      */
  const void* emb;           /* E   [V][r] dtype: parent-token embedding of the head     */
  const void* proj_t;        /* W^T [V][r] dtype: proj_t[v*r + j] = W[j][v]              */
  const float* depth_feat;   /* h   [R][B][r] float32: per-depth head feature            */
  const int32_t* root_token; /* x_t [R]: last verified token, root of the tree           */
  const int32_t* prefix_len; /* [R]: verified-prefix length; position = prefix + depth   */
} pctree_inputs;

/* The emitted tree (Sec. 4.2, App. A).  Nodes are in canonical order: depth
 * ascending, then root-to-node token path lexicographically ascending, so
 * node 0 is the root (token x_t, parent -1, depth 0, logprob 0) and
 * parent[i] < i.  Rows i >= count[r] are padded with token = parent = depth =
 * position = -1 and logprob = -inf (mask rows: zero words).
 *
 * count[r] = -1 marks an abandoned round (see the single-launch exception
 * under the conventions above): then every row of every request is padding
 * and every mask word is zero; nothing of an earlier call's tree remains.
 * The call itself has already returned PCTREE_OK, so a caller that may
 * overlap rounds on one device checks count once the stream has run. */
typedef struct pctree_tree {
  int32_t* token;    /* [R][N] draft token ids                                   */
  int32_t* parent;   /* [R][N] index of the parent node in the same row, -1 root */
  int32_t* depth;    /* [R][N] tree depth (root 0)                               */
  int32_t* position; /* [R][N] prefix_len + depth                                */
  float* logprob;    /* [R][N] joint path score s(c) (Eq. 4), root 0             */
  int32_t* count;    /* [R]    min(N, pool size); 0 for an invalid root; -1 if
                        the round was abandoned (all rows padded)             */
  uint32_t* mask;    /* optional (may be NULL): [R][N][(N+31)/32] ancestor mask,
                        bit j%32 of word j/32 of row i is set iff node j is node
                        i or one of its ancestors (same layout as build_mask)    */
} pctree_tree;

/* Optional per-stage record of the frontier (Alg. 1), for inspection.
 * Entry [r][d][s] describes frontier slot s used at stage d: its token, the
 * slot of its own parent in the frontier of stage d-1 (-1 for the root) and
 * its joint score.  Stage 0 holds the root only.  Unused slots hold
 * (-1, -1, -inf). */
typedef struct pctree_trace {
  int32_t* token;       /* [R][B][k] */
  int32_t* parent_slot; /* [R][B][k] */
  float* score;         /* [R][B][k] */
} pctree_trace;

/* Bytes of workspace that pctree_build_tree and pctree_chain_decode need for
 * `shape` (0 if the shape is invalid or unsupported).  Pure host arithmetic. */
size_t pctree_workspace_bytes(const pctree_shape* shape);

/* Build one round's draft tree for every request (Alg. 1, Eq. 2-4, Sec. 4.2,
 * App. A).  `trace` may be NULL.  The workspace's contents on entry do not
 * matter; on return it holds scratch the caller must not rely on. */
pctree_status pctree_build_tree(const pctree_shape* shape, const pctree_inputs* in,
                                const pctree_tree* out, const pctree_trace* trace,
                                void* workspace, size_t workspace_bytes, void* stream);

/* pctree_build_tree for callers that cannot allocate device memory: code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc.  The same round with the same kernels and results, but its
 * workspace is a fixed array inside the library, PCTREE_NOALLOC_SCRATCH_BYTES
 * bytes per device (each device the library runs on holds its copy until the
 * process ends); the call allocates and frees nothing.  The caller still
 * provides inputs and outputs.  Errors as for pctree_build_tree, plus
 * PCTREE_ERR_WORKSPACE (before any device work) when the shape needs more
 * than PCTREE_NOALLOC_SCRATCH_BYTES of workspace (pctree_workspace_bytes),
 * and PCTREE_ERR_HIP if the array's device address cannot be looked up.
 * Every call on one device shares that device's array: calls whose rounds
 * can overlap on one device (other streams, other host threads) race and
 * corrupt each other; calls ordered on one stream are safe.  Each call
 * clears what it needs before use. */
#define PCTREE_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)
pctree_status pctree_build_tree_noalloc(const pctree_shape* shape, const pctree_inputs* in,
                                        const pctree_tree* out, const pctree_trace* trace,
                                        void* stream);

/* Ancestor-only tree attention mask from parent indices (App. A): row i of
 * request r admits node i and its ancestors.  parent [R][N], count [R] (as
 * emitted by pctree_build_tree), mask [R][N][(N+31)/32] uint32.  Rows at or
 * beyond count are zero.  A parent index that is not in [-1, i) ends that
 * row's walk.  Limits: N <= PCTREE_MAX_MASK_BUDGET. */
pctree_status pctree_build_mask(const int32_t* parent, const int32_t* count, int32_t requests,
                                int32_t budget, uint32_t* mask, void* stream);

/* The DSpark greedy chain of Eq. 1: y_{-1} = x_t, y_d = argmax_v z_d(y_{d-1})
 * (ties to the lowest token id).  Uses vocab, block, rank, requests, dtype and
 * mode of `shape` (topk and budget are ignored; modes PARENT and SHARED give
 * the same chain, INDEPENDENT the chain of argmax_v L_d).  chain_token [R][B+1] gets
 * x_t, y_0..y_{B-1}; chain_logprob [R][B+1] the cumulative log-probabilities
 * (0 for x_t).  Same workspace as pctree_build_tree.  An abandoned round
 * leaves every chain_token entry -1 and every chain_logprob -inf. */
pctree_status pctree_chain_decode(const pctree_shape* shape, const pctree_inputs* in,
                                  int32_t* chain_token, float* chain_logprob, void* workspace,
                                  size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------
 * Verification bookkeeping after a round (Sec. 4.2; App. A, "Tensor
 * implementation").  The emitted tree goes through one target forward, which
 * predicts a greedy next token at every node; these calls turn that into the
 * accepted draft and compact the per-node cache entries.  Same conventions as
 * above (device pointers, asynchronous on `stream`, host-side checks only).
 * W = max_depth + 1 is the width of a row; max_depth is normally B.
 * --------------------------------------------------------------------- */

/* Retrieve indices (App. A): one padded root-to-leaf row per leaf.
 * parent [R][N], count [R] as emitted by pctree_build_tree.  A leaf is a node
 * i < count that is no node's parent; leaf q in ascending node order gets row
 * q of rows [R][N][W]: the node indices from the root down to the leaf,
 * padded with -1.  nrows [R] = number of leaves; rows past it are all -1.
 * Malformed trees do not fault: a parent index outside [0, i) ends the
 * upward walk from node i (that node then heads its row), and a path longer
 * than W keeps its first W nodes from the head.
 * Limits: N <= PCTREE_MAX_MASK_BUDGET, max_depth <= PCTREE_MAX_BLOCK. */
pctree_status pctree_build_retrieve(const int32_t* parent, const int32_t* count, int32_t requests,
                                    int32_t budget, int32_t max_depth, int32_t* rows,
                                    int32_t* nrows, void* stream);

/* Greedy tree acceptance (Sec. 4.2: the standard greedy tree rule; App. A).
 * token [R][N] draft tokens; rows [R][N][W] and nrows [R] from
 * pctree_build_retrieve; target_next [R][N] the target's greedy next token
 * after each node.  Along a row, position l >= 1 is accepted while
 * token[row[l]] == target_next[row[l-1]]; the row accepting the most
 * positions wins (the lowest row on ties).  Outputs per request:
 * accept_len [R] accepted draft tokens (root excluded), accept_row [R] the
 * winning row (-1 if there is none), accept_node [R][W] its accepted node
 * indices from the root, padded with -1, and bonus [R] = target_next at the
 * last accepted node (-1 if there is no row).  A row entry outside [0, N)
 * ends that row.  Limits as for pctree_build_retrieve. */
pctree_status pctree_accept_greedy(const int32_t* token, const int32_t* rows,
                                   const int32_t* nrows, const int32_t* target_next,
                                   int32_t requests, int32_t budget, int32_t max_depth,
                                   int32_t* accept_len, int32_t* accept_row,
                                   int32_t* accept_node, int32_t* bonus, void* stream);

/* Compaction after acceptance (App. A): the cache entries of the accepted
 * row move right after the verified prefix.  `cache` holds, per request and
 * group (e.g. one layer's K or V, or the target hidden states), `capacity`
 * slots of slot_bytes each, contiguous: slot s of group g of request r starts
 * at cache + r*request_stride + g*group_stride + s*slot_bytes.  Tree node i
 * sits at slot prefix_len[r] + i; the accepted nodes n_0..n_a
 * (accept_node [R][W], accept_len [R] from pctree_accept_greedy) move, in
 * place, to slots prefix_len[r] + 0..a.  Other slots keep their contents.
 * A request whose accepted nodes are not strictly increasing, not below N,
 * or reach past `capacity` is left untouched.  slot_bytes, both strides and
 * `cache` must be multiples of 16. */
pctree_status pctree_compact_kv(void* cache, int64_t request_stride, int64_t group_stride,
                                int32_t groups, int32_t capacity, int32_t slot_bytes,
                                const int32_t* prefix_len, const int32_t* accept_node,
                                const int32_t* accept_len, int32_t requests, int32_t budget,
                                int32_t max_depth, void* stream);

/* ---------------------------------------------------------------------
 * Tree-masked verification attention (Sec. 4.2: the packed tree is verified
 * in one target forward; App. A, "Tensor implementation": a node attends to
 * the verified prefix, itself and its root-to-node ancestors).  One
 * attention layer of the target, grouped-query heads, bf16 operands, fp32
 * accumulation and softmax, bf16 output.
 * --------------------------------------------------------------------- */

typedef struct pctree_attn_shape {
  int32_t requests; /* R                                                        */
  int32_t budget;   /* N: tree rows per request, as emitted by the builder      */
  int32_t q_heads;  /* Hq                                                       */
  int32_t kv_heads; /* Hkv, a divisor of Hq; query head h reads kv head h/(Hq/Hkv) */
  int32_t head_dim; /* D: 64 or 128                                             */
  int32_t capacity; /* C: cache slots per request and kv head                   */
  float scale;      /* softmax scale of q.k, > 0, usually 1/sqrt(D)             */
} pctree_attn_shape;

/* Workspace bytes pctree_tree_attention needs for `shape` (0: none, or an
 * invalid shape).  Pure host arithmetic. */
size_t pctree_attention_workspace_bytes(const pctree_attn_shape* shape);

/* out[r][i][h] = sum_s softmax_s(scale * q[r][i][h] . k[r][h/g][s]) v[r][h/g][s]
 * over the admitted slots s of tree node i: the prefix [0, prefix_len[r]) and
 * prefix_len[r] + j for every bit j < count[r] set in mask row i (cache slot
 * prefix_len + j holds tree node j, as after pctree_compact_kv's layout).
 * q [R][N][Hq][D], k_cache and v_cache [R][Hkv][C][D], out [R][N][Hq][D],
 * all bf16 (uint16 bits), 16-byte aligned; mask [R][N][(N+31)/32] as from
 * pctree_build_mask; count [R], prefix_len [R] int32 device arrays.
 * Rows i >= count[r], and rows that admit no slot, are zero.  prefix_len
 * and count are clamped to [0, C] and [0, N], and slots at or past C are
 * never read; slots at or past prefix_len + count are never read either,
 * so they may hold anything.  Admitted slots must hold finite values.
 * Errors: INVALID_ARGUMENT (null or misaligned pointer, size < 1, Hq not a
 * multiple of Hkv, scale not positive and finite), UNSUPPORTED (D not 64 or 128,
 * N > PCTREE_MAX_MASK_BUDGET, R or Hkv > 65535, sizes past the index range),
 * WORKSPACE (a needed workspace null, too small or not 256-byte aligned). */
pctree_status pctree_tree_attention(const pctree_attn_shape* shape, const void* q,
                                    const void* k_cache, const void* v_cache,
                                    const uint32_t* mask, const int32_t* count,
                                    const int32_t* prefix_len, void* out, void* workspace,
                                    size_t workspace_bytes, void* stream);

/* Static, human-readable name of a status code. */
const char* pctree_status_string(pctree_status status);

/* PCTREE_ABI_VERSION of the loaded library. */
int32_t pctree_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* PCTREE_H */
