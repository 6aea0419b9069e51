/*
 * lumo_tree.h - C ABI of the MI355X (gfx950) tree-verification library for the
 * Gated DeltaNet recurrence (LumoTree, arXiv 2609.23900).
 *
 * One speculative-decoding step of a hybrid model's GDN layers, for a batch of
 * requests, each carrying its own candidate tree:
 *   lumo_tree_plan         host: validate parents, derive the tree descriptor
 *   lumo_tree_conv_gather  device: causal conv over each node's ancestry window
 *   lumo_tree_gdn_verify   device: every node's recurrent output from its ancestry
 *   lumo_gdn_commit        device: derive the accepted path, replay it into the
 *                          native state, publish the convolution history
 * plus lumo_tree_attention (the attention layers' tree verification),
 * lumo_draft_select (the drafter's fused argmax / top-k selection), a
 * captured-graph form of the commit, a commit for per-layer history buffers, two
 * deferred verifications in one launch; lumo_tree_gdn_verify_pending and
 * lumo_tree_conv_gather_pending, which fold the publication of one iteration (state
 * replay, conv history) into the verification and convolution of the next, and
 * lumo_tree_gdn_verify_conv_pending, which does both in one pass with the conv outputs
 * never stored; and forms
 * that prepare the operands inside the kernels (lumo_gdn_prep: query/key
 * normalisation, gates from raw inputs).
 *
 * Conventions shared by every entry point
 *   - Device pointers are HIP device (or managed) memory owned by the caller.
 *     The library never allocates or frees device memory on these paths except
 *     the graph object of lumo_gdn_commit_graph_create.
 *   - `stream` is a hipStream_t passed as void* (NULL = the default stream). All
 *     device work is enqueued on it asynchronously, with no host synchronisation,
 *     so every device entry point can be captured into a graph.
 *   - Arguments are validated on the host before anything is enqueued; a non-OK
 *     status means nothing was launched. lumo_last_error() then returns a
 *     description (thread-local, valid until the next call on that thread).
 *   - Calls are stateless and thread-safe.
 *
 * Tensor layouts (rows are physical rows; requests are concatenated, request r
 * owns rows [row_off[r], row_off[r+1]); node i of request r lives at row
 * row_off[r] + slot[i]; rows beyond a request's nodes are padding and are never
 * read or written):
 *   q, k        [n_layers][total_rows][h_k][d_k]            op_dtype
 *   v           [n_layers][total_rows][h_v][d_v]            op_dtype
 *   g, beta     [n_layers][total_rows][h_v]                 float32; alpha = exp(g)
 *   state       [n_req][n_layers][h_v][d_k][d_v]            float32, key-major:
 *                                                           entry (i, j) is R[j][i]
 *   o           [n_layers][total_rows][h_v][d_v]            op_dtype
 *   x, y        [n_layers][total_rows][channels]            op_dtype
 *   conv_hist   [n_req][n_layers][3][channels]              op_dtype, oldest first
 *   w           [n_layers][channels][4]                     float32, tap 3 = newest
 *   bias        [n_layers][channels]                        float32
 * Value head h reads key head h / (h_v / h_k).
 */
#ifndef LUMO_TREE_H
#define LUMO_TREE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    LUMO_OK = 0,
    LUMO_EINVAL = 1,       /* null / misaligned pointer, bad scalar argument      */
    LUMO_EDESC = 2,        /* malformed tree (parents, rows) or plan mismatch     */
    LUMO_ESHAPE = 3,       /* dims inconsistent with each other or with the plan  */
    LUMO_EUNSUPPORTED = 4, /* head size / dtype / option not built                */
    LUMO_EHIP = 5,         /* a HIP call or kernel launch failed                  */
    LUMO_ESPACE = 6        /* caller buffer (plan words, workspace) too small     */
} lumo_status;

typedef enum { LUMO_F32 = 0, LUMO_BF16 = 1 } lumo_dtype;

/* Verification schedules (Sec. IV-A, IV-C). All produce the same outputs. */
typedef enum {
    /* Dependent path groups: the tree is cut into disjoint first-child chains; a
     * chain starts from the pre-tree state (the spine) or from the exported cut
     * state of its parent; chains are launched level by level (one launch per
     * dependency level), each node is updated once. Needs a workspace. */
    LUMO_POLICY_PATHS = 0,
    /* The paper's two launches: the spine exports the cut states of its branch
     * nodes; every other root-to-leaf path then runs from its spine cut state,
     * recomputing off-spine prefixes it shares with other paths. Needs a workspace. */
    LUMO_POLICY_TWO_LEVEL = 1,
    /* Every root-to-leaf path from the pre-tree state in one launch; no cut
     * states, shared prefixes recomputed. No workspace. */
    LUMO_POLICY_RECOMPUTE = 2,
    /* Tree WY form: R_t = gamma_t R0 + sum over ancestors of decayed rank-1
     * terms. With bf16 operands, d_k = d_v = 128 and paths of at most 17 nodes the
     * R0 [K | Q] products run on MFMA (R0 as bf16 hi + lo) and the ancestor-masked
     * triangular system on the vector units; other shapes (fp32 operands, d_k in
     * {16, 32, 64}, d_v below 128, paths of 18 to 32 nodes) run the same form on the
     * vector units in fp32. Paths longer than 32 nodes are refused
     * (LUMO_EUNSUPPORTED). One launch, no workspace, no state dump. Outputs agree
     * with the sequential schedules to rounding, not bitwise. */
    LUMO_POLICY_WY = 3
} lumo_policy;

typedef struct {
    int32_t n_req;    /* requests in the batch                                  */
    int32_t n_layers; /* stacked GDN layers (independent instances)            */
    int32_t h_k;      /* query/key heads                                        */
    int32_t h_v;      /* value heads; h_v % h_k == 0                            */
    int32_t d_k;      /* key dim: 16, 32, 64 or 128                             */
    int32_t d_v;      /* value dim: 16, 32, 64 or 128                           */
    int32_t op_dtype; /* lumo_dtype of q, k, v, o, x, y, conv_hist              */
} lumo_gdn_dims;

/* Host summary of a plan: counts and the word offsets of every section of the
 * int32 plan blob. Filled by lumo_tree_plan; read-only for the caller. */
typedef struct {
    int32_t n_req, total_nodes, total_rows;
    int32_t max_nodes; /* most nodes in one request                           */
    int32_t max_depth; /* most nodes on one root-to-leaf path                 */
    int32_t policy;
    int32_t n_paths;   /* leaves over all requests                            */
    int32_t n_spine;   /* spine nodes over all requests                       */
    int32_t n_seg, n_seg_nodes, n_levels, n_cuts, max_level_seg, max_seg_len;
    int32_t n_words;   /* blob size in int32 words                            */
    /* section offsets (int32 words) inside the blob */
    int32_t o_node_off, o_row_off, o_req, o_parent, o_depth, o_slot, o_row, o_conv_src;
    int32_t o_path_off, o_path_leaf, o_spine_off, o_spine, o_level_off, o_seg, o_seg_nodes;
    int32_t o_dfs, o_dfs_pos;
    /* preorder tables (chunks of 32 preorder positions per request) */
    int32_t n_chunks;    /* chunks over all requests                            */
    int32_t o_pre_row, o_pre_depth, o_pre_ci, o_chunk_off, o_chunk_stack;
    /* attention visibility, per node in slot order */
    int32_t o_vis;
} lumo_plan;

/* A plan whose blob has been copied to device memory. */
typedef struct {
    const int32_t* blob;      /* device copy of the lumo_tree_plan words              */
    const int32_t* host_blob; /* host copy of the same words; read only during a call
                                 (level boundaries of the schedule), never by kernels  */
    lumo_plan plan;           /* the host summary returned with those words           */
} lumo_tree_desc;

/*
 * lumo_tree_plan - validate candidate trees and derive the shared tree descriptor
 * (Sec. III-C; spine-first slots Sec. V-B; path groups Sec. IV-A, Alg. 2; cut
 * states Sec. IV-C, Eq. (4); conv gather sources Sec. V-C).
 *
 *   n_req        requests (>= 0)
 *   node_off     host [n_req+1]: request r owns flat nodes [node_off[r], node_off[r+1])
 *   parent       host [node_off[n_req]]: request-local parent ids; node 0 of a
 *                non-empty request is its root (-1); otherwise 0 <= parent[i] < i
 *   n_rows       host [n_req]: physical rows of request r (>= its node count)
 *   policy       lumo_policy whose schedule the plan carries
 *   blob         host int32 words receiving the plan, or NULL to query the size
 *   blob_words   capacity of blob in words
 *   out          host summary (always filled on LUMO_OK / LUMO_ESPACE)
 *
 * Derived per request (bit-exact, fully determined):
 *   depth (root 0); leaves in increasing id; root-to-leaf paths; spine = the
 *   first-child chain from the root (children ordered by id); slot = physical
 *   order spine first, then the remaining nodes in increasing id; per node the
 *   four conv window sources oldest first (absolute row, or -1-h for committed
 *   history entry h); the verify schedule of `policy`.
 * Blob sections (words; see the o_* offsets):
 *   node_off[n_req+1], row_off[n_req+1], req[N], parent[N], depth[N], slot[N],
 *   row[N] (absolute), conv_src[N][4], path_off[n_req+1], path_leaf[n_paths],
 *   spine_off[n_req+1], spine[n_spine], level_off[n_levels+1],
 *   seg[n_seg][4] = {request, source cut (-1 = pre-tree state), first entry, length},
 *   seg_nodes[n_seg_nodes][3] = {absolute row, writes output (0/1), cut to export (-1 none)},
 *   dfs[N] (per request: node ids in depth-first preorder, children by increasing id),
 *   dfs_pos[N] (position of each node in that order),
 *   pre_row[N], pre_depth[N] (absolute row and depth of the node at each preorder
 *   position), pre_ci[N][4] (16 bytes, little-endian: byte m is the Gram candidate
 *   slot of the node's ancestor at depth m: m when the ancestor precedes the position's
 *   chunk of 32, else 16 + its offset in the chunk; 0xff past the node's depth),
 *   chunk_off[n_req+1],
 *   chunk_stack[n_chunks][16] (rows of the ancestors of each chunk's first node by
 *   depth, -1 beyond its depth),
 *   vis[N][2] (per node in slot order, node_off[r] + slot: its preorder position and
 *   the position one past its subtree; node a is an ancestor-or-self of node i iff
 *   vis[a][0] <= vis[i][0] < vis[a][1]).
 * Returns LUMO_EDESC for malformed trees, LUMO_ESPACE (with out->n_words set)
 * when blob is NULL or too small, LUMO_EINVAL for bad arguments.
 */
lumo_status lumo_tree_plan(int32_t n_req, const int32_t* node_off, const int32_t* parent,
                           const int32_t* n_rows, int32_t policy, int32_t* blob,
                           int64_t blob_words, lumo_plan* out);

/*
 * lumo_tree_gdn_workspace_bytes - device workspace needed by lumo_tree_gdn_verify
 * for this plan: PATHS / TWO_LEVEL one fp32 d_k x d_v matrix per (exported cut,
 * layer, value head) (the cut-state payload of Eq. (4), Sec. IV-C); RECOMPUTE and
 * WY 0.
 */
size_t lumo_tree_gdn_workspace_bytes(const lumo_gdn_dims* dims, const lumo_plan* plan);

/*
 * lumo_tree_conv_gather - tree causal convolution (Sec. V-C, Tab. II row 3).
 * For node i at depth j of request r, layer l, channel c, the window is the last
 * four entries of (conv_hist[r][l][0..2], x along the root-to-i ancestry):
 *   y[l][row(i)][c] = act(bias[l][c] + sum_{t=0..3} w[l][c][t] * window[t][c])
 * accumulated in fp32 in tap order 0..3 starting from the bias, then the
 * activation, then one round-to-nearest-even cast to op_dtype.
 *   channels  multiple of 8; x, y, conv_hist 16-byte aligned
 *   bias      nullable (zero); act 0 = identity, 1 = SiLU
 * Pad rows of y are not written.
 */
lumo_status lumo_tree_conv_gather(const lumo_gdn_dims* dims, const lumo_tree_desc* desc,
                                  int32_t channels, const void* x, const void* conv_hist,
                                  const float* w, const float* bias, int32_t act, void* y,
                                  void* stream);

/*
 * lumo_tree_conv_gather_pending - publish the previous iteration's accepted path into
 * the conv history, then the tree convolution of this iteration from the published
 * history (Alg. 1: publication of iteration t-1 precedes iteration t; Sec. V-C). For
 * every request r and layer l with a valid pending path of length L (1 <= L <=
 * max_path; the previous tree had nodes):
 *   conv_hist[r][l] <- the last three entries of (conv_hist[r][l], x_prev rows of the
 *                      path), in place, exactly as lumo_gdn_commit would publish them;
 *   y               <- lumo_tree_conv_gather from that history.
 * A pending length <= 0 (none, or invalid: -1) or > max_path leaves conv_hist as it is.
 * Requests with no nodes in this iteration are still published. The result equals
 * lumo_gdn_commit's history publication followed by lumo_tree_conv_gather, bit for bit;
 * the commit of the previous iteration is then called with a NULL conv_hist (and NULL
 * x), so that it only derives path_out and path_len.
 *   desc, x, w, bias, act, y   this iteration, as lumo_tree_conv_gather
 *   conv_hist                  in/out [n_req][layers][3][channels]
 *   pend_desc                  the previous iteration's descriptor (same n_req)
 *   max_path, path_out, path_len   as written by that iteration's lumo_gdn_commit
 *   x_prev                     the previous iteration's x, [layers][its rows][channels]
 *                              (nullable when the previous tree had no nodes)
 */
lumo_status lumo_tree_conv_gather_pending(const lumo_gdn_dims* dims, const lumo_tree_desc* desc,
                                          int32_t channels, const void* x, void* conv_hist,
                                          const float* w, const float* bias, int32_t act, void* y,
                                          const lumo_tree_desc* pend_desc, int32_t max_path,
                                          const int32_t* path_out, const int32_t* path_len,
                                          const void* x_prev, void* stream);

/*
 * lumo_gdn_prep - operand preparation inside the kernels (Sec. IV-B: verification
 * takes raw gate inputs and normalises queries and keys itself). Applies to every
 * node of the call (tree nodes, path nodes replayed, pending path nodes).
 *   flags    LUMO_PREP_QK_NORM: every query and key row x (d_k elements) is used as
 *              x / sqrt(sum_i x_i^2 + qk_eps), computed in fp32 from the operands;
 *            LUMO_PREP_RAW_GATES: g and beta hold raw inputs a and b per (node, value
 *              head), and
 *                alpha = exp(-exp(a_log[l][h]) * softplus(a + dt_bias[l][h])),
 *                beta  = 1 / (1 + exp(-b)),
 *              softplus(x) = log(1 + exp(x)), in fp32.
 *   qk_eps   >= 0, finite (LUMO_PREP_QK_NORM)
 *   a_log, dt_bias  device fp32 [n_layers][h_v] (LUMO_PREP_RAW_GATES; else ignored)
 * A NULL lumo_gdn_prep, or flags 0, means the operands are used as given.
 */
#define LUMO_PREP_QK_NORM 1
#define LUMO_PREP_RAW_GATES 2
typedef struct {
    int32_t flags;
    float qk_eps;
    const float* a_log;
    const float* dt_bias;
} lumo_gdn_prep;

/*
 * lumo_tree_gdn_verify - recurrent output of every tree node (Sec. III-B,
 * Eq. (2)-(3); path-parallel scan Sec. IV-A, Alg. 2). For each request r, layer l,
 * value head h and node i, with R_pi the state after the root-to-parent path
 * (R = pre-tree state state0[r][l][h] for the root's parent):
 *   R'_i = alpha_i R_pi;  delta_i = beta_i (v_i - R'_i k_i);
 *   R_i = R'_i + delta_i k_i^T;  o_i = R_i q_i     (alpha_i = exp(g_i))
 * computed with fp32 state and fp32 arithmetic; o is cast once (RNE) to op_dtype.
 *   state0        pre-tree state; never written
 *   o             written at every node row; pad rows untouched
 *   node_states   nullable debug dump [n_layers][total_rows][h_v][d_k][d_v] fp32:
 *                 the state R_i of every node (key-major) at its row. Bitwise equal
 *                 to what lumo_gdn_commit publishes for a path ending at that node.
 *                 Not available with LUMO_POLICY_WY (LUMO_EUNSUPPORTED).
 *   workspace     >= lumo_tree_gdn_workspace_bytes() bytes (nullable when 0)
 *   flags         reserved, must be 0
 * The schedule is the policy the plan was built for.
 */
lumo_status lumo_tree_gdn_verify(const lumo_gdn_dims* dims, const lumo_tree_desc* desc,
                                 const void* q, const void* k, const void* v, const float* g,
                                 const float* beta, const float* state0, void* o,
                                 float* node_states, void* workspace, size_t workspace_bytes,
                                 int32_t flags, void* stream);

/*
 * lumo_tree_gdn_verify_prep - lumo_tree_gdn_verify with the operands prepared as
 * `prep` says (nullable; Sec. IV-B). Takes a plan built for LUMO_POLICY_WY (paths of
 * at most 32 nodes, the shapes of that policy) or LUMO_POLICY_RECOMPUTE (the
 * sequential scan of every path from the pre-tree state: any supported shape, either
 * operand type, any depth; bitwise what lumo_gdn_commit_prep publishes for the same
 * path); plans that export cut states to a workspace (PATHS, TWO_LEVEL) are refused
 * with LUMO_EUNSUPPORTED, as this call takes no workspace. No node-state dump.
 */
lumo_status lumo_tree_gdn_verify_prep(const lumo_gdn_dims* dims, const lumo_tree_desc* desc,
                                      const lumo_gdn_prep* prep, const void* q, const void* k,
                                      const void* v, const float* g, const float* beta,
                                      const float* state0, void* o, void* stream);

/*
 * lumo_tree_gdn_verify_pending - publish the previous iteration's accepted path into
 * the state bank and verify this iteration's tree from the published state, in one
 * pass over the state (Alg. 1: publication of iteration t-1 precedes verification of
 * iteration t; deferred into this call, each state tile is read once and written once
 * instead of being read twice and written once). For every request r, layer l and
 * value head h:
 *   state[r][l][h] <- the state after replaying the pending path of r with the
 *                     update of lumo_gdn_commit and the pending operands, in place;
 *   o              <- as lumo_tree_gdn_verify with state0 = that published state.
 *   desc, q, k, v, g, beta, o   this iteration; desc's plan must use LUMO_POLICY_WY
 *                               (bf16 operands, d_k = d_v = 128, paths of at most
 *                               17 nodes), else LUMO_EUNSUPPORTED
 *   state                       in/out: the state bank before the pending publication
 *   pend_desc                   the previous iteration's descriptor (same n_req)
 *   max_path, path_out, path_len  as written by lumo_gdn_commit for pend_desc;
 *                               path_len[r] <= 0 leaves request r's state as it is
 *   pend_k, pend_v, pend_g, pend_beta  the previous iteration's operands (device,
 *                               rows of pend_desc)
 *   prep                        nullable; operand preparation of both iterations
 * The replay sums its dot products in another order than lumo_gdn_commit, so the
 * published state agrees with it to fp32 rounding, not bitwise. Requests with no
 * nodes in this iteration are still published.
 */
lumo_status lumo_tree_gdn_verify_pending(const lumo_gdn_dims* dims, const lumo_tree_desc* desc,
                                         const lumo_gdn_prep* prep, const void* q, const void* k, const void* v,
                                         const float* g, const float* beta, float* state, void* o,
                                         const lumo_tree_desc* pend_desc, int32_t max_path,
                                         const int32_t* path_out, const int32_t* path_len,
                                         const void* pend_k, const void* pend_v,
                                         const float* pend_g, const float* pend_beta, void* stream);

/*
 * lumo_tree_gdn_verify_pending_pair - two lumo_tree_gdn_verify_pending calls in one
 * launch (Sec. IV-B: each layer runs its own update; Alg. 1: a layer's state is
 * published before that layer's next verification reads it). Each call is described by
 * a lumo_gdn_pending_call holding exactly the arguments of lumo_tree_gdn_verify_pending
 * and gives the same results, bit for bit. The point is a model calling the step layer
 * by layer: call a verifies layer l (its path published earlier: pend_desc of a batch
 * without nodes, so that nothing is pending) while call b publishes the pending path
 * into layer l + 1's state bank (desc of a batch without nodes: nothing to verify);
 * the two run side by side on the device, so the publication costs the layer call
 * little time.
 *   a    required; b nullable (then this is call a alone)
 * Both calls run the 32-column form (four waves of 32 state columns per value head,
 * the same bits as any other launch of the call). Host errors as for
 * lumo_tree_gdn_verify_pending, per call; LUMO_EUNSUPPORTED when the two calls differ
 * in query/key normalisation (LUMO_PREP_QK_NORM). The calls must not write the same
 * memory (outputs, state banks); a call's pending path may be shared.
 */
typedef struct {
    const lumo_gdn_dims* dims;
    const lumo_tree_desc* desc;
    const lumo_gdn_prep* prep;
    const void* q;
    const void* k;
    const void* v;
    const float* g;
    const float* beta;
    float* state;
    void* o;
    const lumo_tree_desc* pend_desc;
    int32_t max_path;
    const int32_t* path_out;
    const int32_t* path_len;
    const void* pend_k;
    const void* pend_v;
    const float* pend_g;
    const float* pend_beta;
} lumo_gdn_pending_call;
lumo_status lumo_tree_gdn_verify_pending_pair(const lumo_gdn_pending_call* a, const lumo_gdn_pending_call* b,
                                              void* stream);

/*
 * lumo_tree_gdn_verify_conv_pending - lumo_tree_conv_gather_pending and
 * lumo_tree_gdn_verify_pending in one pass, with the conv outputs never stored (Sec.
 * V-C: windows gathered from the history and the candidate inputs, the tap computation
 * fused, tap order and cast points kept; each output is rounded to bf16 where the
 * separate conv stores it, then used as the verification's operand): the tree causal
 * conv of x (channels q | k | v, window = the node's three nearest
 * ancestors after the history, taps and activation as lumo_tree_conv_gather) gives
 * each node's query, key and value rows; the pending path's keys and values are the
 * same conv of x_prev along the path (from the history before its publication); the
 * history is published from the pending path; the state bank receives the pending
 * path's replay and the tree is verified from it, as lumo_tree_gdn_verify_pending.
 * Results equal the two calls in sequence with y split into q, k, v (bit for bit).
 *   channels   2 h_k d_k + h_v d_v; x channel 0 .. h_k d_k - 1 are the queries (key
 *              head hk at hk d_k), then the keys, then the values (value head h at
 *              2 h_k d_k + h d_v)
 *   x          [n_layers][total_rows][channels] bf16, this iteration's rows
 *   conv_hist  [n_req][n_layers][3][channels] bf16, read, and written in place where a
 *              path is pending
 *   w, bias, act   as lumo_tree_conv_gather (bias nullable); the layer's weights, so
 *              the pending path's keys and values are convolved with them as well
 *   g, beta, state, o, prep   as lumo_tree_gdn_verify_pending
 *   pend_desc, max_path, path_out, path_len, pend_g, pend_beta   as
 *              lumo_tree_gdn_verify_pending; x_prev is the previous iteration's x
 *              ([n_layers][its total_rows][channels])
 * Needs h_v = 2 h_k and the plan and dims of lumo_tree_gdn_verify_pending, else
 * LUMO_EUNSUPPORTED; LUMO_ESHAPE for another channel count. Every request's history
 * slice and state tile are read and written by one block, so calls must not overlap
 * with other users of conv_hist or state.
 */
lumo_status lumo_tree_gdn_verify_conv_pending(const lumo_gdn_dims* dims, const lumo_tree_desc* desc,
                                              const lumo_gdn_prep* prep, int32_t channels, const void* x,
                                              void* conv_hist, const float* w, const float* bias,
                                              int32_t act, const float* g, const float* beta, float* state,
                                              void* o, const lumo_tree_desc* pend_desc, int32_t max_path,
                                              const int32_t* path_out, const int32_t* path_len,
                                              const void* x_prev, const float* pend_g,
                                              const float* pend_beta, void* stream);


/*
 * lumo_gdn_commit - publish the accepted path (Alg. 1 publication; Alg. 2 replay;
 * device-selected path Sec. V-A; conv history Sec. V-C).
 *   accepted_node  device [n_req]: request-local accepted node, -1 = none
 *   max_path       fixed path capacity (1..4096); the work shape depends only on it
 *   path_out       device [n_req][max_path]: root-first accepted path, padded -1
 *   path_len       device [n_req]: its length; -1 when accepted_node[r] is not in
 *                  [-1, nodes of r) or the path is longer than max_path (then the
 *                  state and history of request r are left unchanged)
 *   k, v, g, beta  the operands recorded for verification (q is not needed)
 *   state          in/out: the pre-tree state, replaced in place by the state after
 *                  replaying the path with the update of lumo_tree_gdn_verify
 *                  (bitwise the same arithmetic); untouched for an empty path.
 *                  NULL defers the replay to the next lumo_tree_gdn_verify_pending
 *                  (k, v, g, beta may then be NULL too): only path_out, path_len and
 *                  the conv history are written
 *   x, conv_hist   nullable pair: when given, conv_hist[r][l] becomes the last
 *                  three entries of (conv_hist[r][l], x rows of the path), in place;
 *                  NULL leaves that publication to the next
 *                  lumo_tree_conv_gather_pending
 */
lumo_status lumo_gdn_commit(const lumo_gdn_dims* dims, const lumo_tree_desc* desc,
                            int32_t max_path, const int32_t* accepted_node, int32_t* path_out,
                            int32_t* path_len, const void* k, const void* v, const float* g,
                            const float* beta, float* state, int32_t channels, const void* x,
                            void* conv_hist, void* stream);

/*
 * lumo_gdn_commit_hist_layers - lumo_gdn_commit's path derivation and conv-history
 * publication (Alg. 1 publication; device-selected path Sec. V-A; conv history Sec. V-C)
 * for models that keep each layer's buffers apart and call the verification layer by
 * layer (Sec. IV-B: every layer runs its own update kernel). One launch publishes the
 * accepted path into the history of every layer; each layer's state is left to its
 * next lumo_tree_gdn_verify_pending (deferred replay), and its conv then runs as
 * lumo_tree_conv_gather on the published history.
 *   dims, desc, max_path, accepted_node, path_out, path_len   as lumo_gdn_commit
 *                  (dims->n_layers layers, at most 128, else LUMO_EUNSUPPORTED)
 *   channels       positive multiple of 8 (LUMO_ESHAPE)
 *   x_layers       HOST array of n_layers device pointers: layer l's x of this
 *                  iteration, [total_rows][channels] of op_dtype (16-byte aligned;
 *                  entries may be NULL when the tree has no nodes)
 *   conv_hist_layers  HOST array of n_layers device pointers: layer l's history,
 *                  [n_req][3][channels] of op_dtype (16-byte aligned), in/out:
 *                  conv_hist_layers[l][r] becomes the last three entries of
 *                  (conv_hist_layers[l][r], x_layers[l] rows of the path), in place
 * The tables are read on the host during the call (the pointers are passed to the
 * kernel by value), so they may be freed or reused when it returns. path_out, path_len
 * and every history equal what lumo_gdn_commit writes with the same layers stacked,
 * bit for bit; empty and invalid paths leave the histories unchanged. Histories of
 * different layers must not overlap.
 */
lumo_status lumo_gdn_commit_hist_layers(const lumo_gdn_dims* dims, const lumo_tree_desc* desc,
                                        int32_t max_path, const int32_t* accepted_node,
                                        int32_t* path_out, int32_t* path_len, int32_t channels,
                                        const void* const* x_layers, void* const* conv_hist_layers,
                                        void* stream);

/*
 * lumo_gdn_commit_prep - lumo_gdn_commit whose replay uses the operands prepared as
 * `prep` says (nullable; any plan policy). The replay then agrees with a verification
 * given the same `prep` to fp32 rounding.
 */
lumo_status lumo_gdn_commit_prep(const lumo_gdn_dims* dims, const lumo_tree_desc* desc,
                                 const lumo_gdn_prep* prep, int32_t max_path,
                                 const int32_t* accepted_node, int32_t* path_out,
                                 int32_t* path_len, const void* k, const void* v, const float* g,
                                 const float* beta, float* state, int32_t channels,
                                 const void* x, void* conv_hist, void* stream);

/*
 * Tree attention (Sec. V-B; visibility Sec. III-A): the attention layers' verification
 * of the same candidate tree. Query row i (a tree node) attends to its request's
 * committed context and to the tree nodes on its own root-to-node path, itself
 * included; pad rows are invisible:
 *   s_j = scale (q_i . k_j),  o_i = sum_j exp(s_j - lse_i) v_j,  lse_i = log sum_j exp(s_j)
 * over those keys j. Query head h reads key/value head h / (h_q / h_kv).
 *   lumo_attn_dims  n_req; h_q, h_kv with h_q / h_kv in {1, 2, 4, 8}; d = 128;
 *                   op_dtype = LUMO_BF16
 *   q           [total_rows][h_q][d] at the tree's physical rows (spine first)
 *   k_tree, v_tree  [total_rows][h_kv][d], the tree nodes' own keys and values at the
 *               same rows (spine-contiguous)
 *   k_ctx, v_ctx    [tokens][h_kv][d]; request r's context is tokens
 *               ctx_off[r] .. ctx_off[r+1]-1 (ctx_off device int32 [n_req+1])
 *   max_ctx     host, >= every request's context length
 *   scale       softmax scale (> 0)
 *   o           [total_rows][h_q][d] op_dtype, written at node rows only
 *   lse         [total_rows][h_q] fp32 natural log, written at node rows only
 *   n_split     context partitions reduced separately and combined (split-K), >= 1;
 *               lumo_tree_attention_splits suggests one that fills the device
 *   workspace   >= lumo_tree_attention_workspace_bytes(dims, plan, n_split) bytes
 * Keys are reduced context first (partition by partition), then the tree nodes in
 * physical slot order; the reduction order is fixed for given shapes and n_split.
 * All pointers 16-byte aligned; LUMO_EUNSUPPORTED for other shapes.
 */
typedef struct {
    int32_t n_req, h_q, h_kv, d, op_dtype;
} lumo_attn_dims;

size_t lumo_tree_attention_workspace_bytes(const lumo_attn_dims* dims, const lumo_plan* plan,
                                           int32_t n_split);
int32_t lumo_tree_attention_splits(const lumo_attn_dims* dims, const lumo_plan* plan, int32_t max_ctx);
lumo_status lumo_tree_attention(const lumo_attn_dims* dims, const lumo_tree_desc* desc,
                                const int32_t* ctx_off, int32_t max_ctx, float scale,
                                const void* q, const void* k_ctx, const void* v_ctx,
                                const void* k_tree, const void* v_tree, void* o, float* lse,
                                int32_t n_split, void* workspace, size_t workspace_bytes,
                                void* stream);

/*
 * lumo_tree_attention_noalloc - lumo_tree_attention for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc): the partial results of the key ranges go to a fixed scratch array
 * of LUMO_TREE_ATTENTION_SCRATCH_BYTES (32 MiB) that the library holds on each device it
 * runs on until the process ends, instead of a caller workspace. Same arguments and
 * results as lumo_tree_attention otherwise (bitwise, for the same n_split); it calls no
 * allocating routine. LUMO_ESPACE, before any launch, when
 * lumo_tree_attention_workspace_bytes(dims, plan, n_split) exceeds the array (at d =
 * 128: (n_split + 1) x total_rows x h_q <= 65,027). Every call on one device shares
 * that device's array: calls that overlap in time on one device (two streams, two
 * threads) race and must be ordered by the caller. The first call on a device, with
 * that device current, looks up the array's device address.
 */
#define LUMO_TREE_ATTENTION_SCRATCH_BYTES (32u << 20)
lumo_status lumo_tree_attention_noalloc(const lumo_attn_dims* dims, const lumo_tree_desc* desc,
                                        const int32_t* ctx_off, int32_t max_ctx, float scale,
                                        const void* q, const void* k_ctx, const void* v_ctx,
                                        const void* k_tree, const void* v_tree, void* o, float* lse,
                                        int32_t n_split, void* stream);

/*
 * Fused draft selection (Sec. V-D): from one full-vocabulary logits row per drafting
 * position, the principal (spine) token and k ordered sibling candidates in one pass.
 * The two reference operations break ties differently, and both are reproduced:
 *   spine[r]       the lowest index among the maximal logits of row r (argmax)
 *   cand[r][0..k)  the k indices ranked first: logit descending; among equal logits
 *                  index ascending (ties = 0) or descending (ties = 1) (top-k). The
 *                  spine token may also appear among the candidates.
 * A NaN logit (any payload) ranks above every number, NaNs equal among themselves;
 * -0 equals +0. The result is exact (an ordering of the stored values), independent of
 * n_split.
 *   logits      device, row r at element r * ld, `vocab` logits each; float32
 *               (dtype LUMO_F32) or bfloat16 bit patterns (LUMO_BF16); 16-byte aligned.
 *               Elements between rows (ld > vocab) are never used.
 *   rows >= 0, vocab >= 1, ld >= vocab, 1 <= k <= min(8, vocab), ties 0 or 1
 *   spine       device int32 [rows];  cand  device int32 [rows][k]
 *   n_split     parts each row is cut into (1..4096); lumo_draft_select_splits
 *               suggests one for the row count and vocabulary. With n_split > 1 the
 *               parts are reduced separately (each by four wavefronts) and merged by a
 *               second kernel.
 *   workspace   device, >= lumo_draft_select_workspace_bytes(rows, k, n_split)
 *               bytes, 16-byte aligned (0 and NULL allowed when n_split = 1). No
 *               initial contents are needed; calls that share a workspace must not
 *               overlap in time.
 * LUMO_EUNSUPPORTED for k > 8.
 */
size_t lumo_draft_select_workspace_bytes(int32_t rows, int32_t k, int32_t n_split);
int32_t lumo_draft_select_splits(int32_t rows, int32_t vocab, int32_t dtype);
lumo_status lumo_draft_select(int32_t rows, int32_t vocab, int64_t ld, int32_t dtype, int32_t k,
                              int32_t ties, const void* logits, int32_t* spine, int32_t* cand,
                              int32_t n_split, void* workspace, size_t workspace_bytes,
                              void* stream);

/* Opaque captured commit: the fixed-shape committer graph of Sec. V-A. */
typedef struct lumo_commit_graph lumo_commit_graph;

/*
 * lumo_gdn_commit_graph_create - the fixed-shape committer of Sec. V-A (Alg. 1
 * publication): capture the launches of lumo_gdn_commit with these exact arguments
 * into an instantiated HIP graph, so that one replay per serving iteration derives the
 * device-selected path, replays it into the native state and publishes the conv
 * history with no host path list. The work shape depends only on max_path. `prep`
 * (nullable) prepares the replayed operands as lumo_gdn_commit_prep does (Sec. IV-B:
 * the recorded keys normalised, the gates from raw inputs); its a_log and dt_bias are
 * bound by address too. Device buffers are bound by address: replays read the current
 * contents of accepted_node (and every operand) at launch time. The caller keeps all buffers alive until
 * destroy. Errors: the validation of lumo_gdn_commit, before any capture; LUMO_EHIP
 * when capture or instantiation fails (nothing is left captured).
 */
lumo_status lumo_gdn_commit_graph_create(const lumo_gdn_dims* dims, const lumo_tree_desc* desc,
                                         const lumo_gdn_prep* prep, int32_t max_path,
                                         const int32_t* accepted_node,
                                         int32_t* path_out, int32_t* path_len, const void* k,
                                         const void* v, const float* g, const float* beta,
                                         float* state, int32_t channels, const void* x,
                                         void* conv_hist, lumo_commit_graph** out);

/* Replay the captured commit (Sec. V-A) on `stream`; LUMO_EINVAL for a NULL graph,
 * LUMO_EHIP when the launch fails. */
lumo_status lumo_gdn_commit_graph_launch(lumo_commit_graph* graph, void* stream);

/* Release the graph (NULL is ignored). */
void lumo_gdn_commit_graph_destroy(lumo_commit_graph* graph);

/* Description of the last non-OK status returned on this thread ("" if none). */
const char* lumo_last_error(void);

/* Library version string. */
const char* lumo_version(void);

#ifdef __cplusplus
}
#endif

#endif /* LUMO_TREE_H */
