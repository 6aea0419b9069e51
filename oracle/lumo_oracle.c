/*
 * Plain fp64 CPU oracle for tree verification of the Gated DeltaNet recurrence.
 *
 * TEST INFRASTRUCTURE ONLY. Only the test suite, the smoke check and the CPU
 * baseline leg of the benchmark load this library. The GPU library never links,
 * includes or calls it, and it shares no code with the GPU library.
 *
 * What it computes (LumoTree, arXiv 2609.23900):
 *   - Sec. III-B, Eq. (2)-(3): for one head, R in R^{d_v x d_k}; a node i with
 *     parent pi(i), decay alpha_i and write strength beta_i applies
 *         R'_i   = alpha_i R_pi(i)
 *         delta_i = beta_i (v_i - R'_i k_i)
 *         R_i    = R'_i + delta_i k_i^T
 *         o_i    = R_i q_i
 *     and every node consumes the state of exactly its root-to-parent path
 *     (Sec. III-A). The oracle walks parent[] from each node to the root and
 *     replays the whole ancestry from the pre-tree state, one node at a time,
 *     in fp64. No caching, no reordering, no blocking.
 *   - Alg. 1 / Alg. 2 replay: the accepted path is replayed from the pre-tree
 *     state with the same update and the resulting state is published.
 *   - Sec. V-C: the causal convolution of a node sees the committed history
 *     followed by the inputs along its ancestry (path predecessors, not adjacent
 *     packed rows); the window is the last four entries, taps applied oldest to
 *     newest.
 *
 *   - Sec. V-B tree attention: every query row sees the committed context and its
 *     own ancestry (plain two-pass softmax in fp64, orc_tree_attention).
 *   - Sec. V-D draft selection: the argmax (spine) token and the ordered top-k
 *     candidates of a logits row, with their two tie conventions (orc_draft_select).
 *   - Sec. IV-B operand preparation (optional, prep_flags): verification takes raw
 *     gate inputs and normalises queries and keys itself. With ORC_PREP_QK_NORM
 *     every query and key row x is used as x / sqrt(|x|^2 + qk_eps); with
 *     ORC_PREP_RAW_GATES the g and beta arrays hold raw inputs a and b and
 *         alpha = exp(-exp(A_log[l][h]) * softplus(a + dt_bias[l][h])),
 *         beta  = 1 / (1 + exp(-b)),
 *     the Gated DeltaNet gate parametrisation. The replay uses the same prepared
 *     operands.
 *
 * Readings where the paper is silent (gate parametrisation alpha = exp(g), the
 * root is itself an updated node, tap order, SiLU activation, history length 3,
 * the normalisation constant) are listed in the design notes of the repository.
 *
 * Layouts (physical rows; row of a node = absolute row index):
 *   q, k [layers][rows][h_k][d_k]; v [layers][rows][h_v][d_v];
 *   g, beta [layers][rows][h_v] float32;
 *   state [requests][layers][h_v][d_k][d_v] float32, key-major: element
 *   (key i, value j) of head matrix R (R[j][i]) is stored at i*d_v + j.
 *   Operands are float32 (dtype 0) or bfloat16 bit patterns (dtype 1).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

typedef struct {
    int n_req, n_layers, h_k, h_v, d_k, d_v;
    int op_dtype;      /* 0 = float32, 1 = bfloat16 bit patterns */
    int total_rows;
    int gate_is_alpha; /* 0: g holds log(alpha); 1: g holds alpha itself (exact hand tests) */
    int prep_flags;    /* ORC_PREP_QK_NORM | ORC_PREP_RAW_GATES (Sec. IV-B), 0 = none */
    double qk_eps;     /* ORC_PREP_QK_NORM: added to |x|^2 under the square root */
    const float* a_log;   /* ORC_PREP_RAW_GATES: [layers][h_v] */
    const float* dt_bias; /* ORC_PREP_RAW_GATES: [layers][h_v] */
} orc_dims;

enum { ORC_PREP_QK_NORM = 1, ORC_PREP_RAW_GATES = 2 };

/* Sec. IV-B: a query or key row divided by the square root of (its squared norm + eps). */
static void qk_prepare(const orc_dims* d, double* x, int n) {
    if (!(d->prep_flags & ORC_PREP_QK_NORM)) return;
    double ss = 0.0;
    for (int i = 0; i < n; ++i) ss += x[i] * x[i];
    const double scale = sqrt(ss + d->qk_eps);
    for (int i = 0; i < n; ++i) x[i] /= scale;
}

/* Decay and write strength of one (node, value head) from its g and beta entries. */
static void gates(const orc_dims* d, int l, int h, double g_in, double b_in, double* alpha, double* beta) {
    if (d->prep_flags & ORC_PREP_RAW_GATES) {
        const long lh = (long)l * d->h_v + h;
        const double x = g_in + (double)d->dt_bias[lh];
        const double softplus = (x > 0.0 ? x : 0.0) + log1p(exp(-fabs(x)));  /* log(1 + e^x) */
        *alpha = exp(-exp((double)d->a_log[lh]) * softplus);
        *beta = 1.0 / (1.0 + exp(-b_in));
    } else {
        *alpha = d->gate_is_alpha ? g_in : exp(g_in);
        *beta = b_in;
    }
}

/* Decode one operand element to double. bfloat16 is the upper half of a float32. */
static double ld_op(const void* base, long idx, int dtype) {
    if (dtype == 0) return (double)((const float*)base)[idx];
    uint32_t bits = ((uint32_t)((const uint16_t*)base)[idx]) << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

/* Root-first ancestry of `node` (request-local ids). Returns its length, or -1 on a
 * malformed parent array (cycle / out of range / longer than cap). */
static int ancestry(const int* parent, int n_nodes, int node, int* out, int cap) {
    int len = 0;
    for (int x = node; x >= 0; x = parent[x]) {
        if (x >= n_nodes || len >= cap) return -1;
        out[len++] = x;
    }
    for (int a = 0, b = len - 1; a < b; ++a, --b) {
        int t = out[a];
        out[a] = out[b];
        out[b] = t;
    }
    return len;
}

/* Load the pre-tree state of (r, l, h) into R (value-major, d_v x d_k). */
static void load_state(const orc_dims* d, const float* state, int r, int l, int h, double* R) {
    const long base = ((((long)r * d->n_layers + l) * d->h_v + h) * d->d_k) * (long)d->d_v;
    for (int i = 0; i < d->d_k; ++i)
        for (int j = 0; j < d->d_v; ++j) R[(long)j * d->d_k + i] = (double)state[base + (long)i * d->d_v + j];
}

static void store_state(const orc_dims* d, const double* R, double* out /* [d_k][d_v] */) {
    for (int i = 0; i < d->d_k; ++i)
        for (int j = 0; j < d->d_v; ++j) out[(long)i * d->d_v + j] = R[(long)j * d->d_k + i];
}

/* Eq. (2)-(3) for the node stored at physical row `row`, layer l, value head h. */
static void gdn_node_update(const orc_dims* d, double* R, double* Rk, double* kv, double* vv,
                            int l, int row, int h, const void* k, const void* v, const float* g,
                            const float* beta) {
    const int dk = d->d_k, dv = d->d_v;
    const int hk = h / (d->h_v / d->h_k);
    const long kb = (((long)l * d->total_rows + row) * d->h_k + hk) * dk;
    const long vb = (((long)l * d->total_rows + row) * d->h_v + h) * dv;
    const long gb = ((long)l * d->total_rows + row) * d->h_v + h;
    double a, b;
    gates(d, l, h, (double)g[gb], (double)beta[gb], &a, &b);
    for (int i = 0; i < dk; ++i) kv[i] = ld_op(k, kb + i, d->op_dtype);
    qk_prepare(d, kv, dk);
    for (int j = 0; j < dv; ++j) vv[j] = ld_op(v, vb + j, d->op_dtype);
    /* R' = alpha R */
    for (long e = 0; e < (long)dv * dk; ++e) R[e] *= a;
    /* delta = beta (v - R' k);  R = R' + delta k^T */
    for (int j = 0; j < dv; ++j) {
        double s = 0.0;
        for (int i = 0; i < dk; ++i) s += R[(long)j * dk + i] * kv[i];
        Rk[j] = b * (vv[j] - s);
    }
    for (int j = 0; j < dv; ++j)
        for (int i = 0; i < dk; ++i) R[(long)j * dk + i] += Rk[j] * kv[i];
}

/* o = R q for the query stored at `row`. */
static void gdn_output(const orc_dims* d, const double* R, int l, int row, int h, const void* q,
                       double* qv, double* o) {
    const int dk = d->d_k, dv = d->d_v;
    const int hk = h / (d->h_v / d->h_k);
    const long qb = (((long)l * d->total_rows + row) * d->h_k + hk) * dk;
    for (int i = 0; i < dk; ++i) qv[i] = ld_op(q, qb + i, d->op_dtype);
    qk_prepare(d, qv, dk);
    for (int j = 0; j < dv; ++j) {
        double s = 0.0;
        for (int i = 0; i < dk; ++i) s += R[(long)j * dk + i] * qv[i];
        o[j] = s;
    }
}

typedef struct {
    double *R, *Rk, *kv, *vv, *qv;
    int* path;
} scratch_t;

static int scratch_alloc(const orc_dims* d, int cap, scratch_t* s) {
    s->R = (double*)malloc(sizeof(double) * (size_t)d->d_k * d->d_v);
    s->Rk = (double*)malloc(sizeof(double) * (size_t)d->d_v);
    s->kv = (double*)malloc(sizeof(double) * (size_t)d->d_k);
    s->vv = (double*)malloc(sizeof(double) * (size_t)d->d_v);
    s->qv = (double*)malloc(sizeof(double) * (size_t)d->d_k);
    s->path = (int*)malloc(sizeof(int) * (size_t)(cap > 0 ? cap : 1));
    return (s->R && s->Rk && s->kv && s->vv && s->qv && s->path) ? 0 : -1;
}

static void scratch_free(scratch_t* s) {
    free(s->R);
    free(s->Rk);
    free(s->kv);
    free(s->vv);
    free(s->qv);
    free(s->path);
}

/*
 * Output (and optionally state) of selected nodes of one (request, layer, value head).
 *   parent[n_nodes]: request-local parent ids (-1 root); row[n_nodes]: absolute rows.
 *   o_out [n_targets][d_v]; state_out [n_targets][d_k][d_v] (key-major) or NULL.
 * Returns 0, or -1 on a malformed tree / allocation failure.
 */
int orc_verify_nodes(const orc_dims* d, int n_nodes, const int* parent, const int* row, int r,
                     int l, int h, int n_targets, const int* targets, const void* q, const void* k,
                     const void* v, const float* g, const float* beta, const float* state0,
                     double* o_out, double* state_out) {
    scratch_t s;
    if (scratch_alloc(d, n_nodes, &s)) {
        scratch_free(&s);
        return -1;
    }
    int rc = 0;
    for (int t = 0; t < n_targets && rc == 0; ++t) {
        const int len = ancestry(parent, n_nodes, targets[t], s.path, n_nodes);
        if (len < 0) {
            rc = -1;
            break;
        }
        load_state(d, state0, r, l, h, s.R);
        for (int p = 0; p < len; ++p)
            gdn_node_update(d, s.R, s.Rk, s.kv, s.vv, l, row[s.path[p]], h, k, v, g, beta);
        gdn_output(d, s.R, l, row[targets[t]], h, q, s.qv, o_out + (long)t * d->d_v);
        if (state_out) store_state(d, s.R, state_out + (long)t * d->d_k * d->d_v);
    }
    scratch_free(&s);
    return rc;
}

/*
 * All outputs of all requests: o_all [layers][rows][h_v][d_v] in fp64 (rows that hold
 * no node are left untouched). node_off[n_req+1] splits the flat parent/row arrays.
 * Work over (request, layer, head) instances is spread over n_threads threads.
 */
int orc_verify_all(const orc_dims* d, const int* node_off, const int* parent, const int* row,
                   const void* q, const void* k, const void* v, const float* g,
                   const float* beta, const float* state0, double* o_all, int n_threads) {
    const long n_inst = (long)d->n_req * d->n_layers * d->h_v;
    int bad = 0;
#ifdef _OPENMP
#pragma omp parallel for schedule(dynamic, 1) num_threads(n_threads > 0 ? n_threads : 1) reduction(| : bad)
#endif
    for (long inst = 0; inst < n_inst; ++inst) {
        const int h = (int)(inst % d->h_v);
        const int l = (int)((inst / d->h_v) % d->n_layers);
        const int r = (int)(inst / ((long)d->h_v * d->n_layers));
        const int n = node_off[r + 1] - node_off[r];
        const int* par = parent + node_off[r];
        const int* rw = row + node_off[r];
        double* o = (double*)malloc(sizeof(double) * (size_t)d->d_v);
        if (!o) {
            bad |= 1;
            continue;
        }
        for (int i = 0; i < n; ++i) {
            if (orc_verify_nodes(d, n, par, rw, r, l, h, 1, &i, q, k, v, g, beta, state0, o, NULL)) {
                bad |= 1;
                break;
            }
            double* dst = o_all + (((long)l * d->total_rows + rw[i]) * d->h_v + h) * d->d_v;
            memcpy(dst, o, sizeof(double) * (size_t)d->d_v);
        }
        free(o);
    }
    (void)n_threads;
    return bad ? -1 : 0;
}

/*
 * Accepted-path replay (Alg. 1 publication, Alg. 2 replay) for all instances.
 *   accepted[n_req]: request-local accepted node, -1 = none (empty replay).
 *   path_out[n_req][max_path]: root-first node ids padded with -1; path_len[n_req].
 *   An accepted node outside [-1, nodes of r), or a path longer than max_path, is a
 *   selection that names no publishable path: path_len[r] = -1, path_out[r] all -1,
 *   and request r's state is published unchanged (the paper publishes only a path it
 *   accepted; the report of -1 is this interface's convention).
 *   state_in: pre-tree state; state_out: published state (fp64, same layout).
 * Returns 0, or -1 when a parent array is malformed.
 */
int orc_commit(const orc_dims* d, const int* node_off, const int* parent, const int* row,
               const int* accepted, int max_path, const void* k, const void* v, const float* g,
               const float* beta, const float* state_in, double* state_out, int* path_out,
               int* path_len, int n_threads) {
    int bad = 0;
    for (int r = 0; r < d->n_req; ++r) {
        const int n = node_off[r + 1] - node_off[r];
        int* po = path_out + (long)r * max_path;
        for (int p = 0; p < max_path; ++p) po[p] = -1;
        path_len[r] = 0;
        if (accepted[r] == -1) continue;
        if (accepted[r] < -1 || accepted[r] >= n) {
            path_len[r] = -1;
            continue;
        }
        int* tmp = (int*)malloc(sizeof(int) * (size_t)(n > 0 ? n : 1));
        const int len = ancestry(parent + node_off[r], n, accepted[r], tmp, n);
        if (len < 0) {
            free(tmp);
            return -1;
        }
        if (len > max_path) {
            path_len[r] = -1;
            free(tmp);
            continue;
        }
        for (int p = 0; p < len; ++p) po[p] = tmp[p];
        path_len[r] = len;
        free(tmp);
    }
    const long n_inst = (long)d->n_req * d->n_layers * d->h_v;
#ifdef _OPENMP
#pragma omp parallel for schedule(dynamic, 1) num_threads(n_threads > 0 ? n_threads : 1) reduction(| : bad)
#endif
    for (long inst = 0; inst < n_inst; ++inst) {
        const int h = (int)(inst % d->h_v);
        const int l = (int)((inst / d->h_v) % d->n_layers);
        const int r = (int)(inst / ((long)d->h_v * d->n_layers));
        scratch_t s;
        if (scratch_alloc(d, 1, &s)) {
            scratch_free(&s);
            bad |= 1;
            continue;
        }
        const int* rw = row + node_off[r];
        load_state(d, state_in, r, l, h, s.R);
        for (int p = 0; p < path_len[r]; ++p)
            gdn_node_update(d, s.R, s.Rk, s.kv, s.vv, l, rw[path_out[(long)r * max_path + p]], h, k, v,
                            g, beta);
        const long base = ((((long)r * d->n_layers + l) * d->h_v + h) * d->d_k) * (long)d->d_v;
        store_state(d, s.R, state_out + base);
        scratch_free(&s);
    }
    (void)n_threads;
    return bad ? -1 : 0;
}

/*
 * Tree causal convolution (Sec. V-C) of every node, every layer:
 *   seq(i) = hist[0], hist[1], hist[2], x[row(a_0)], ..., x[row(a_j)]   (a_0 root, a_j = i)
 *   window = last four entries of seq(i), oldest first
 *   y[l][row(i)][c] = act(bias[l][c] + sum_{t=0..3} w[l][c][t] * window[t][c])
 * act: 0 identity, 1 SiLU (x * sigmoid(x)). bias may be NULL (zero).
 * x, y [layers][rows][C]; hist [requests][layers][3][C]; w [layers][C][4].
 */
int orc_conv_all(int n_req, int n_layers, int total_rows, int channels, int op_dtype,
                 const int* node_off, const int* parent, const int* row, const void* x,
                 const void* hist, const float* w, const float* bias, int act, double* y) {
    for (int r = 0; r < n_req; ++r) {
        const int n = node_off[r + 1] - node_off[r];
        const int* par = parent + node_off[r];
        const int* rw = row + node_off[r];
        int* path = (int*)malloc(sizeof(int) * (size_t)(n > 0 ? n : 1));
        for (int i = 0; i < n; ++i) {
            const int len = ancestry(par, n, i, path, n);
            if (len < 0) {
                free(path);
                return -1;
            }
            for (int l = 0; l < n_layers; ++l) {
                for (int c = 0; c < channels; ++c) {
                    double acc = bias ? (double)bias[(long)l * channels + c] : 0.0;
                    for (int t = 0; t < 4; ++t) {
                        /* position in seq: hist occupies 0..2, ancestry 3..3+len-1 */
                        const int pos = 3 + len - 4 + t;
                        double xv;
                        if (pos >= 3)
                            xv = ld_op(x, ((long)l * total_rows + rw[path[pos - 3]]) * channels + c, op_dtype);
                        else
                            xv = ld_op(hist, (((long)r * n_layers + l) * 3 + pos) * channels + c, op_dtype);
                        acc += (double)w[((long)l * channels + c) * 4 + t] * xv;
                    }
                    if (act == 1) acc = acc / (1.0 + exp(-acc));
                    y[((long)l * total_rows + rw[i]) * channels + c] = acc;
                }
            }
        }
        free(path);
    }
    return 0;
}

/*
 * Convolution-history publication for the accepted path (Alg. 1):
 *   hist'[r][l] = last three entries of (hist[r][l][0..2], x[row(a_0)], ..., x[row(a_{L-1})]).
 * path[n_req][max_path] root-first, path_len[n_req]. hist_out in fp64.
 */
int orc_conv_hist_publish(int n_req, int n_layers, int total_rows, int channels, int op_dtype,
                          const int* node_off, const int* row, const int* path, const int* path_len,
                          int max_path, const void* x, const void* hist, double* hist_out) {
    for (int r = 0; r < n_req; ++r) {
        const int L = path_len[r];
        const int* rw = row + node_off[r];
        for (int l = 0; l < n_layers; ++l)
            for (int e = 0; e < 3; ++e) {
                const int pos = L + e; /* entry e of the last three of a (3 + L)-long sequence */
                for (int c = 0; c < channels; ++c) {
                    double val;
                    if (pos < 3)
                        val = ld_op(hist, (((long)r * n_layers + l) * 3 + pos) * channels + c, op_dtype);
                    else
                        val = ld_op(x, ((long)l * total_rows + rw[path[(long)r * max_path + pos - 3]]) * channels + c,
                                    op_dtype);
                    hist_out[(((long)r * n_layers + l) * 3 + e) * channels + c] = val;
                }
            }
    }
    return 0;
}

/*
 * Tree attention (Sec. V-B; Sec. III-A visibility): query row i of request r sees the
 * request's committed context (tokens ctx_off[r] .. ctx_off[r+1]-1) and the tree nodes
 * on its own root-to-node path, itself included; pad rows are invisible. For query head
 * h (key/value head h / (h_q / h_kv)):
 *   s_j = scale * (q_i . k_j)  over the visible keys j,
 *   o_i = sum_j exp(s_j - lse) v_j,  lse = log sum_j exp(s_j).
 * q [rows][h_q][d]; k_tree, v_tree [rows][h_kv][d] at the tree's physical rows;
 * k_ctx, v_ctx [tokens][h_kv][d]. o [rows][h_q][d] and lse [rows][h_q] in fp64 (rows
 * that hold no node are left untouched). Returns 0, or -1 on a malformed tree.
 */
int orc_tree_attention(int n_req, int h_q, int h_kv, int d, int op_dtype, const int* node_off,
                       const int* parent, const int* row, const int* ctx_off, double scale,
                       const void* q, const void* k_ctx, const void* v_ctx, const void* k_tree,
                       const void* v_tree, double* o, double* lse, int n_threads) {
    int bad = 0;
    const int grp = h_q / h_kv;
    const long n_all = node_off[n_req];
    /* one (request, node) per iteration; r is found by scanning node_off */
#ifdef _OPENMP
#pragma omp parallel for schedule(dynamic, 1) num_threads(n_threads > 0 ? n_threads : 1) reduction(| : bad)
#endif
    for (long flat = 0; flat < n_all; ++flat) {
        int r = 0;
        while (node_off[r + 1] <= flat) ++r;
        const int i = (int)(flat - node_off[r]);
        const int n = node_off[r + 1] - node_off[r];
        const int* par = parent + node_off[r];
        const int* rw = row + node_off[r];
        const long c0 = ctx_off[r], nc = ctx_off[r + 1] - ctx_off[r];
        int* path = (int*)malloc(sizeof(int) * (size_t)n);
        double* sc = (double*)malloc(sizeof(double) * (size_t)(nc + n + 1));
        double* acc = (double*)malloc(sizeof(double) * (size_t)d);
        const int len = (path && sc && acc) ? ancestry(par, n, i, path, n) : -1;
        if (len < 0) {
            bad |= 1;
        } else {
            for (int h = 0; h < h_q; ++h) {
                const int hk = h / grp;
                const long qb = ((long)rw[i] * h_q + h) * d;
                /* scores: context first, then the path root first */
                double mx = -INFINITY;
                for (long t = 0; t < nc + len; ++t) {
                    const void* kk = t < nc ? k_ctx : k_tree;
                    const long kb = t < nc ? ((c0 + t) * h_kv + hk) * d : ((long)rw[path[t - nc]] * h_kv + hk) * d;
                    double s = 0.0;
                    for (int e = 0; e < d; ++e) s += ld_op(q, qb + e, op_dtype) * ld_op(kk, kb + e, op_dtype);
                    sc[t] = scale * s;
                    if (sc[t] > mx) mx = sc[t];
                }
                double sum = 0.0;
                for (int e = 0; e < d; ++e) acc[e] = 0.0;
                for (long t = 0; t < nc + len; ++t) {
                    const double w = exp(sc[t] - mx);
                    sum += w;
                    const void* vv = t < nc ? v_ctx : v_tree;
                    const long vb = t < nc ? ((c0 + t) * h_kv + hk) * d : ((long)rw[path[t - nc]] * h_kv + hk) * d;
                    for (int e = 0; e < d; ++e) acc[e] += w * ld_op(vv, vb + e, op_dtype);
                }
                for (int e = 0; e < d; ++e) o[qb + e] = acc[e] / sum;
                lse[(long)rw[i] * h_q + h] = mx + log(sum);
            }
        }
        free(path);
        free(sc);
        free(acc);
    }
    (void)n_threads;
    return bad ? -1 : 0;
}

/*
 * Fused draft selection (Sec. V-D): from one full-vocabulary logits row the principal
 * (spine) token and k ordered sibling candidates, two outputs whose reference
 * operations break ties differently:
 *   spine[r]      = the lowest index among the maximal logits of row r (argmax);
 *   cand[r][0..k) = the k indices ranked first by logit, descending, and among equal
 *                   logits by index: ascending (ties = 0) or descending (ties = 1)
 *                   (top-k). The spine token may appear among the candidates.
 * A NaN logit ranks above every number (NaNs equal among themselves); -0 equals +0.
 * Plain definition: one scan for the spine, then k selection passes over the row,
 * each taking the best index not yet taken.
 * logits [rows][vocab], float32 (dtype 0) or bfloat16 bit patterns (dtype 1).
 */
static int sel_greater(double a, double b) { /* a ranks strictly above b by value */
    if (isnan(a)) return !isnan(b);
    if (isnan(b)) return 0;
    return a > b;
}

static int sel_before(double a, int ia, double b, int ib, int ties) {
    if (sel_greater(a, b)) return 1;
    if (sel_greater(b, a)) return 0;
    return ties == 0 ? ia < ib : ia > ib;
}

int orc_draft_select(int rows, int vocab, int k, int op_dtype, int ties, const void* logits, int* spine,
                     int* cand, int n_threads) {
    if (k < 1 || k > vocab || (ties != 0 && ties != 1)) return 1;
#ifdef _OPENMP
#pragma omp parallel for schedule(dynamic, 1) num_threads(n_threads > 0 ? n_threads : 1)
#endif
    for (int r = 0; r < rows; ++r) {
        const long base = (long)r * vocab;
        int best = 0;
        for (int i = 1; i < vocab; ++i)
            if (sel_greater(ld_op(logits, base + i, op_dtype), ld_op(logits, base + best, op_dtype))) best = i;
        spine[r] = best;
        for (int j = 0; j < k; ++j) {
            int pick = -1;
            for (int i = 0; i < vocab; ++i) {
                int taken = 0;
                for (int m = 0; m < j; ++m)
                    if (cand[(long)r * k + m] == i) taken = 1;
                if (taken) continue;
                if (pick < 0 || sel_before(ld_op(logits, base + i, op_dtype), i,
                                           ld_op(logits, base + pick, op_dtype), pick, ties))
                    pick = i;
            }
            cand[(long)r * k + j] = pick;
        }
    }
    return 0;
}

int orc_max_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
