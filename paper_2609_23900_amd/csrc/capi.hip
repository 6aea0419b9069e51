// C ABI of the library: host-side validation, dispatch to the kernel launchers,
// captured commit graphs, and error reporting. No exception crosses this boundary.
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>

#include "internal.h"
#include "commit.h"
#include "launch.h"
#include "verify_wy.h"
#include "select.h"

#include <algorithm>

namespace lumo {

namespace {
thread_local std::string g_err;
}

lumo_status fail(lumo_status st, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return st;
}

void clear_error() { g_err.clear(); }

namespace {

bool pow2_head(int d) { return d == 16 || d == 32 || d == 64 || d == 128; }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

lumo_status check_ptr(const void* p, const char* fn, const char* name, bool nullable = false) {
    if (!p) return nullable ? LUMO_OK : fail(LUMO_EINVAL, "%s: %s is NULL", fn, name);
    if (!aligned16(p)) return fail(LUMO_EINVAL, "%s: %s is not 16-byte aligned", fn, name);
    return LUMO_OK;
}

#define LUMO_TRY(expr)                      \
    do {                                    \
        lumo_status st_ = (expr);           \
        if (st_ != LUMO_OK) return st_;     \
    } while (0)

lumo_status check_dims(const lumo_gdn_dims* d, const char* fn) {
    if (!d) return fail(LUMO_EINVAL, "%s: dims is NULL", fn);
    if (d->n_req < 0 || d->n_layers < 1 || d->h_k < 1 || d->h_v < 1)
        return fail(LUMO_ESHAPE, "%s: need n_req >= 0 and n_layers, h_k, h_v >= 1", fn);
    if (d->h_v % d->h_k) return fail(LUMO_ESHAPE, "%s: h_v (%d) is not a multiple of h_k (%d)", fn, d->h_v, d->h_k);
    if (!pow2_head(d->d_k) || !pow2_head(d->d_v))
        return fail(LUMO_EUNSUPPORTED, "%s: d_k=%d d_v=%d (supported: 16, 32, 64, 128)", fn, d->d_k, d->d_v);
    if (d->op_dtype != LUMO_F32 && d->op_dtype != LUMO_BF16)
        return fail(LUMO_EUNSUPPORTED, "%s: op_dtype %d", fn, d->op_dtype);
    return LUMO_OK;
}

// The matrix-core WY kernel's shape limits (bf16, d_k = d_v = 128, at most kWyMaxDepth
// nodes per path): the deferred publication and the fused conv live in it.
lumo_status check_wy(const lumo_gdn_dims* d, const lumo_tree_desc* desc, const char* fn) {
    if (desc->plan.policy != LUMO_POLICY_WY)
        return fail(LUMO_EUNSUPPORTED, "%s: needs a plan built for LUMO_POLICY_WY (plan policy %d)", fn,
                    desc->plan.policy);
    if (d->op_dtype != LUMO_BF16 || d->d_k != 128 || d->d_v != 128)
        return fail(LUMO_EUNSUPPORTED, "%s: built for bf16 operands with d_k = d_v = 128", fn);
    if (desc->plan.max_depth > kWyMaxDepth)
        return fail(LUMO_EUNSUPPORTED, "%s: handles paths of at most %d nodes (plan has %d)", fn, kWyMaxDepth,
                    desc->plan.max_depth);
    return LUMO_OK;
}

// A WY plan's verification: the matrix-core kernel for its shapes, the vector-ALU WY
// kernel for the others (any supported d_k, d_v and operand type; paths of at most
// kWyvMaxDepth nodes).
lumo_status check_wy_verify(const lumo_gdn_dims* d, const lumo_tree_desc* desc, const char* fn) {
    if (desc->plan.policy != LUMO_POLICY_WY)
        return fail(LUMO_EUNSUPPORTED, "%s: needs a plan built for LUMO_POLICY_WY (plan policy %d)", fn,
                    desc->plan.policy);
    if (!wy_mfma_shape(*d, desc->plan) && desc->plan.max_depth > kWyvMaxDepth)
        return fail(LUMO_EUNSUPPORTED, "%s: the WY policy handles paths of at most %d nodes (plan has %d)", fn,
                    kWyvMaxDepth, desc->plan.max_depth);
    return LUMO_OK;
}

hipError_t launch_wy_any(const lumo_gdn_dims& d, const lumo_tree_desc& desc, const GdnArgs& a, hipStream_t s) {
    return wy_mfma_shape(d, desc.plan) ? launch_wy(d, desc, a, s) : launch_wyv(d, desc, a, s);
}

// Operand preparation: flags, constant and gate parameters; NULL means none.
lumo_status check_prep(const lumo_gdn_prep* prep, const char* fn, PrepArgs& out) {
    out = PrepArgs{};
    if (!prep) return LUMO_OK;
    if (prep->flags & ~(LUMO_PREP_QK_NORM | LUMO_PREP_RAW_GATES))
        return fail(LUMO_EINVAL, "%s: prep flags 0x%x (known: QK_NORM 1, RAW_GATES 2)", fn, prep->flags);
    if ((prep->flags & LUMO_PREP_QK_NORM) && !(prep->qk_eps >= 0.f && prep->qk_eps <= 3.0e38f))
        return fail(LUMO_EINVAL, "%s: prep qk_eps must be finite and >= 0", fn);
    if (prep->flags & LUMO_PREP_RAW_GATES) {
        if (!prep->a_log || !prep->dt_bias) return fail(LUMO_EINVAL, "%s: raw gates need a_log and dt_bias", fn);
        if ((reinterpret_cast<uintptr_t>(prep->a_log) | reinterpret_cast<uintptr_t>(prep->dt_bias)) & 3u)
            return fail(LUMO_EINVAL, "%s: a_log and dt_bias must be 4-byte aligned", fn);
    }
    out.flags = prep->flags;
    out.qk_eps = prep->qk_eps;
    out.a_log = prep->a_log;
    out.dt_bias = prep->dt_bias;
    return LUMO_OK;
}

lumo_status check_desc(const lumo_gdn_dims* d, const lumo_tree_desc* desc, const char* fn) {
    if (!desc) return fail(LUMO_EINVAL, "%s: desc is NULL", fn);
    const lumo_plan& p = desc->plan;
    if (p.n_req != d->n_req)
        return fail(LUMO_EDESC, "%s: plan has %d requests, dims %d", fn, p.n_req, d->n_req);
    if (p.n_words <= 0 || p.total_nodes < 0 || p.total_rows < p.total_nodes)
        return fail(LUMO_EDESC, "%s: malformed plan summary", fn);
    if (!desc->blob || !desc->host_blob) return fail(LUMO_EINVAL, "%s: desc blob pointers are NULL", fn);
    if (p.o_seg_nodes + kSegNodeWords * (int64_t)p.n_seg_nodes > p.n_words)
        return fail(LUMO_EDESC, "%s: plan offsets exceed its size", fn);
    return LUMO_OK;
}

}  // namespace
}  // namespace lumo

using namespace lumo;

extern "C" const char* lumo_last_error(void) { return g_err.c_str(); }

extern "C" const char* lumo_version(void) { return "lumo_tree 0.1 gfx950"; }

extern "C" size_t lumo_tree_gdn_workspace_bytes(const lumo_gdn_dims* d, const lumo_plan* p) {
    if (!d || !p) return 0;
    if (p->policy != LUMO_POLICY_PATHS && p->policy != LUMO_POLICY_TWO_LEVEL) return 0;
    return (size_t)p->n_cuts * d->n_layers * d->h_v * d->d_k * d->d_v * sizeof(float);
}

extern "C" lumo_status lumo_tree_conv_gather(const lumo_gdn_dims* dims, const lumo_tree_desc* desc,
                                             int32_t channels, const void* x, const void* conv_hist,
                                             const float* w, const float* bias, int32_t act, void* y,
                                             void* stream) {
    static const char* fn = "lumo_tree_conv_gather";
    clear_error();
    LUMO_TRY(check_dims(dims, fn));
    LUMO_TRY(check_desc(dims, desc, fn));
    if (channels <= 0 || channels % 8) return fail(LUMO_ESHAPE, "%s: channels %d must be a positive multiple of 8", fn, channels);
    if (act != 0 && act != 1) return fail(LUMO_EINVAL, "%s: act %d (0 identity, 1 SiLU)", fn, act);
    if (desc->plan.total_nodes == 0) return LUMO_OK;
    LUMO_TRY(check_ptr(x, fn, "x"));
    LUMO_TRY(check_ptr(conv_hist, fn, "conv_hist"));
    LUMO_TRY(check_ptr(w, fn, "w"));
    LUMO_TRY(check_ptr(bias, fn, "bias", true));
    LUMO_TRY(check_ptr(y, fn, "y"));
    ConvArgs a{channels, x, conv_hist, w, bias, act, y};
    hipError_t e = launch_conv(*dims, *desc, a, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return fail(LUMO_EHIP, "%s: launch failed: %s", fn, hipGetErrorString(e));
    return LUMO_OK;
}

extern "C" lumo_status lumo_tree_conv_gather_pending(const lumo_gdn_dims* dims, const lumo_tree_desc* desc,
                                                     int32_t channels, const void* x, void* conv_hist,
                                                     const float* w, const float* bias, int32_t act, void* y,
                                                     const lumo_tree_desc* pend_desc, int32_t max_path,
                                                     const int32_t* path_out, const int32_t* path_len,
                                                     const void* x_prev, void* stream) {
    static const char* fn = "lumo_tree_conv_gather_pending";
    clear_error();
    LUMO_TRY(check_dims(dims, fn));
    LUMO_TRY(check_desc(dims, desc, fn));
    if (!pend_desc) return fail(LUMO_EINVAL, "%s: pend_desc is NULL", fn);
    LUMO_TRY(check_desc(dims, pend_desc, fn));
    if (channels <= 0 || channels % 8) return fail(LUMO_ESHAPE, "%s: channels %d must be a positive multiple of 8", fn, channels);
    if (act != 0 && act != 1) return fail(LUMO_EINVAL, "%s: act %d (0 identity, 1 SiLU)", fn, act);
    if (max_path < 1 || max_path > 4096) return fail(LUMO_EINVAL, "%s: max_path %d (1..4096)", fn, max_path);
    if (dims->n_req == 0) return LUMO_OK;
    LUMO_TRY(check_ptr(conv_hist, fn, "conv_hist"));
    LUMO_TRY(check_ptr(path_out, fn, "path_out"));
    LUMO_TRY(check_ptr(path_len, fn, "path_len"));
    if (pend_desc->plan.total_nodes > 0) LUMO_TRY(check_ptr(x_prev, fn, "x_prev"));
    if (desc->plan.total_nodes > 0) {
        LUMO_TRY(check_ptr(x, fn, "x"));
        LUMO_TRY(check_ptr(w, fn, "w"));
        LUMO_TRY(check_ptr(bias, fn, "bias", true));
        LUMO_TRY(check_ptr(y, fn, "y"));
    }
    ConvArgs a{channels, x, conv_hist, w, bias, act, y};
    ConvPendArgs pa{pend_desc, max_path, path_out, path_len, x_prev};
    hipError_t e = launch_conv(*dims, *desc, a, static_cast<hipStream_t>(stream), &pa);
    if (e != hipSuccess) return fail(LUMO_EHIP, "%s: launch failed: %s", fn, hipGetErrorString(e));
    return LUMO_OK;
}

extern "C" lumo_status lumo_tree_gdn_verify(const lumo_gdn_dims* dims, const lumo_tree_desc* desc, const void* q,
                                            const void* k, const void* v, const float* g, const float* beta,
                                            const float* state0, void* o, float* node_states, void* workspace,
                                            size_t workspace_bytes, int32_t flags, void* stream) {
    static const char* fn = "lumo_tree_gdn_verify";
    clear_error();
    LUMO_TRY(check_dims(dims, fn));
    LUMO_TRY(check_desc(dims, desc, fn));
    if (flags != 0) return fail(LUMO_EINVAL, "%s: flags must be 0", fn);
    const int policy = desc->plan.policy;
    if (policy < LUMO_POLICY_PATHS || policy > LUMO_POLICY_WY) return fail(LUMO_EDESC, "%s: plan policy %d", fn, policy);
    if (desc->plan.total_nodes == 0) return LUMO_OK;
    LUMO_TRY(check_ptr(q, fn, "q"));
    LUMO_TRY(check_ptr(k, fn, "k"));
    LUMO_TRY(check_ptr(v, fn, "v"));
    LUMO_TRY(check_ptr(g, fn, "g"));
    LUMO_TRY(check_ptr(beta, fn, "beta"));
    LUMO_TRY(check_ptr(state0, fn, "state0"));
    LUMO_TRY(check_ptr(o, fn, "o"));
    LUMO_TRY(check_ptr(node_states, fn, "node_states", true));
    if (policy == LUMO_POLICY_WY) {
        if (node_states) return fail(LUMO_EUNSUPPORTED, "%s: the WY policy keeps no per-node states", fn);
        LUMO_TRY(check_wy_verify(dims, desc, fn));
    }
    const size_t need = lumo_tree_gdn_workspace_bytes(dims, &desc->plan);
    if (need) {
        LUMO_TRY(check_ptr(workspace, fn, "workspace"));
        if (workspace_bytes < need)
            return fail(LUMO_ESPACE, "%s: workspace needs %zu bytes, got %zu", fn, need, workspace_bytes);
    }
    GdnArgs a{q, k, v, g, beta, state0, o, node_states, static_cast<float*>(workspace)};
    hipError_t e;
    if (policy == LUMO_POLICY_WY) {
        e = launch_wy_any(*dims, *desc, a, static_cast<hipStream_t>(stream));
    } else {
        e = launch_scan(*dims, *desc, a, static_cast<hipStream_t>(stream));
    }
    if (e == hipErrorNotSupported) return fail(LUMO_EUNSUPPORTED, "%s: policy %d not compiled into the library", fn, policy);
    if (e != hipSuccess) return fail(LUMO_EHIP, "%s: launch failed: %s", fn, hipGetErrorString(e));
    return LUMO_OK;
}

extern "C" lumo_status lumo_tree_gdn_verify_prep(const lumo_gdn_dims* dims, const lumo_tree_desc* desc,
                                                 const lumo_gdn_prep* prep, const void* q, const void* k,
                                                 const void* v, const float* g, const float* beta,
                                                 const float* state0, void* o, void* stream) {
    static const char* fn = "lumo_tree_gdn_verify_prep";
    clear_error();
    LUMO_TRY(check_dims(dims, fn));
    LUMO_TRY(check_desc(dims, desc, fn));
    const int policy = desc->plan.policy;
    if (policy == LUMO_POLICY_PATHS || policy == LUMO_POLICY_TWO_LEVEL)
        return fail(LUMO_EUNSUPPORTED,
                    "%s: plan policy %d exports cut states to a workspace, which this call does not take "
                    "(use LUMO_POLICY_RECOMPUTE or LUMO_POLICY_WY)", fn, policy);
    if (policy != LUMO_POLICY_RECOMPUTE) LUMO_TRY(check_wy_verify(dims, desc, fn));
    PrepArgs pr;
    LUMO_TRY(check_prep(prep, fn, pr));
    if (desc->plan.total_nodes == 0) return LUMO_OK;
    LUMO_TRY(check_ptr(q, fn, "q"));
    LUMO_TRY(check_ptr(k, fn, "k"));
    LUMO_TRY(check_ptr(v, fn, "v"));
    LUMO_TRY(check_ptr(g, fn, "g"));
    LUMO_TRY(check_ptr(beta, fn, "beta"));
    LUMO_TRY(check_ptr(state0, fn, "state0"));
    LUMO_TRY(check_ptr(o, fn, "o"));
    GdnArgs a{q, k, v, g, beta, state0, o, nullptr, nullptr, pr};
    hipError_t e = policy == LUMO_POLICY_WY ? launch_wy_any(*dims, *desc, a, static_cast<hipStream_t>(stream))
                                            : launch_scan(*dims, *desc, a, static_cast<hipStream_t>(stream));
    if (e == hipErrorNotSupported) return fail(LUMO_EUNSUPPORTED, "%s: not compiled into the library", fn);
    if (e != hipSuccess) return fail(LUMO_EHIP, "%s: launch failed: %s", fn, hipGetErrorString(e));
    return LUMO_OK;
}

namespace {

// Host validation of a deferred verification (lumo_tree_gdn_verify_pending); fills the
// launch arguments. LUMO_OK with *empty set when there is nothing to launch.
lumo_status check_pending(const lumo_gdn_dims* dims, const lumo_tree_desc* desc, const lumo_gdn_prep* prep,
                          const void* q, const void* k, const void* v, const float* g, const float* beta, float* state,
                          void* o, const lumo_tree_desc* pend_desc, int32_t max_path, const int32_t* path_out,
                          const int32_t* path_len, const void* pend_k, const void* pend_v, const float* pend_g,
                          const float* pend_beta, const char* fn, GdnArgs& a, PendArgs& pa, bool& empty) {
    LUMO_TRY(check_dims(dims, fn));
    LUMO_TRY(check_desc(dims, desc, fn));
    if (!pend_desc) return fail(LUMO_EINVAL, "%s: pend_desc is NULL", fn);
    LUMO_TRY(check_desc(dims, pend_desc, fn));
    LUMO_TRY(check_wy(dims, desc, fn));
    PrepArgs pr;
    LUMO_TRY(check_prep(prep, fn, pr));
    if (max_path < 1 || max_path > 4096) return fail(LUMO_EINVAL, "%s: max_path %d (1..4096)", fn, max_path);
    empty = dims->n_req == 0;
    if (empty) return LUMO_OK;
    LUMO_TRY(check_ptr(state, fn, "state"));
    LUMO_TRY(check_ptr(path_out, fn, "path_out"));
    LUMO_TRY(check_ptr(path_len, fn, "path_len"));
    if (pend_desc->plan.total_nodes > 0) {
        LUMO_TRY(check_ptr(pend_k, fn, "pend_k"));
        LUMO_TRY(check_ptr(pend_v, fn, "pend_v"));
        LUMO_TRY(check_ptr(pend_g, fn, "pend_g"));
        LUMO_TRY(check_ptr(pend_beta, fn, "pend_beta"));
    }
    if (desc->plan.total_nodes > 0) {
        LUMO_TRY(check_ptr(q, fn, "q"));
        LUMO_TRY(check_ptr(k, fn, "k"));
        LUMO_TRY(check_ptr(v, fn, "v"));
        LUMO_TRY(check_ptr(g, fn, "g"));
        LUMO_TRY(check_ptr(beta, fn, "beta"));
        LUMO_TRY(check_ptr(o, fn, "o"));
    }
    a = GdnArgs{q, k, v, g, beta, state, o, nullptr, nullptr, pr};
    pa = PendArgs{pend_desc, max_path, path_out, path_len, pend_k, pend_v, pend_g, pend_beta, state};
    return LUMO_OK;
}

}  // namespace

extern "C" lumo_status lumo_tree_gdn_verify_pending(const lumo_gdn_dims* dims, const lumo_tree_desc* desc,
                                                    const lumo_gdn_prep* prep,
                                                    const void* q, const void* k, const void* v, const float* g,
                                                    const float* beta, float* state, void* o,
                                                    const lumo_tree_desc* pend_desc, int32_t max_path,
                                                    const int32_t* path_out, const int32_t* path_len,
                                                    const void* pend_k, const void* pend_v, const float* pend_g,
                                                    const float* pend_beta, void* stream) {
    static const char* fn = "lumo_tree_gdn_verify_pending";
    clear_error();
    GdnArgs a;
    PendArgs pa;
    bool empty = false;
    LUMO_TRY(check_pending(dims, desc, prep, q, k, v, g, beta, state, o, pend_desc, max_path, path_out, path_len,
                           pend_k, pend_v, pend_g, pend_beta, fn, a, pa, empty));
    if (empty) return LUMO_OK;
    hipError_t e = launch_wy(*dims, *desc, a, static_cast<hipStream_t>(stream), &pa);
    if (e == hipErrorNotSupported) return fail(LUMO_EUNSUPPORTED, "%s: not compiled into the library", fn);
    if (e != hipSuccess) return fail(LUMO_EHIP, "%s: launch failed: %s", fn, hipGetErrorString(e));
    return LUMO_OK;
}

extern "C" lumo_status lumo_tree_gdn_verify_pending_pair(const lumo_gdn_pending_call* ca,
                                                         const lumo_gdn_pending_call* cb, void* stream) {
    static const char* fn = "lumo_tree_gdn_verify_pending_pair";
    clear_error();
    if (!ca) return fail(LUMO_EINVAL, "%s: call a is NULL", fn);
    const lumo_gdn_pending_call* c[2] = {ca, cb};
    GdnArgs a[2];
    PendArgs pa[2];
    bool empty[2] = {true, true};
    for (int i = 0; i < 2; ++i) {
        if (!c[i]) continue;
        LUMO_TRY(check_pending(c[i]->dims, c[i]->desc, c[i]->prep, c[i]->q, c[i]->k, c[i]->v, c[i]->g, c[i]->beta,
                               c[i]->state, c[i]->o, c[i]->pend_desc, c[i]->max_path, c[i]->path_out,
                               c[i]->path_len, c[i]->pend_k, c[i]->pend_v, c[i]->pend_g, c[i]->pend_beta, fn, a[i],
                               pa[i], empty[i]));
    }
    if (empty[0] && empty[1]) return LUMO_OK;
    if (!empty[0] && !empty[1] &&
        ((a[0].prep.flags & LUMO_PREP_QK_NORM) != 0) != ((a[1].prep.flags & LUMO_PREP_QK_NORM) != 0))
        return fail(LUMO_EUNSUPPORTED, "%s: both calls must take the same query/key normalisation", fn);
    // a call without requests contributes no blocks: it takes the other call's arguments
    const int i0 = empty[0] ? 1 : 0, i1 = empty[1] ? 0 : 1;
    lumo_gdn_dims d0 = *c[i0]->dims, d1 = *c[i1]->dims;
    if (empty[0]) d0.n_req = 0;
    if (empty[1]) d1.n_req = 0;
    hipError_t e = launch_wy_pair(d0, *c[i0]->desc, a[i0], pa[i0], d1, *c[i1]->desc, a[i1], pa[i1],
                                  static_cast<hipStream_t>(stream));
    if (e == hipErrorNotSupported)
        return fail(LUMO_EUNSUPPORTED, "%s: trees deeper than the WY form's limit", fn);
    if (e != hipSuccess) return fail(LUMO_EHIP, "%s: launch failed: %s", fn, hipGetErrorString(e));
    return LUMO_OK;
}

extern "C" lumo_status lumo_tree_gdn_verify_conv_pending(
    const lumo_gdn_dims* dims, const lumo_tree_desc* desc, const lumo_gdn_prep* prep, int32_t channels, const void* x,
    void* conv_hist, const float* w, const float* bias, int32_t act, const float* g, const float* beta, float* state,
    void* o, const lumo_tree_desc* pend_desc, int32_t max_path, const int32_t* path_out, const int32_t* path_len,
    const void* x_prev, const float* pend_g, const float* pend_beta, void* stream) {
    static const char* fn = "lumo_tree_gdn_verify_conv_pending";
    clear_error();
    LUMO_TRY(check_dims(dims, fn));
    LUMO_TRY(check_desc(dims, desc, fn));
    if (!pend_desc) return fail(LUMO_EINVAL, "%s: pend_desc is NULL", fn);
    LUMO_TRY(check_desc(dims, pend_desc, fn));
    LUMO_TRY(check_wy(dims, desc, fn));
    PrepArgs pr;
    LUMO_TRY(check_prep(prep, fn, pr));
    if (dims->h_v != 2 * dims->h_k)
        return fail(LUMO_EUNSUPPORTED, "%s: h_v / h_k = 2 only (got %d / %d)", fn, dims->h_v, dims->h_k);
    if (channels != 2 * dims->h_k * dims->d_k + dims->h_v * dims->d_v)
        return fail(LUMO_ESHAPE, "%s: channels %d, expected 2 h_k d_k + h_v d_v = %d", fn, channels,
                    2 * dims->h_k * dims->d_k + dims->h_v * dims->d_v);
    if (act != 0 && act != 1) return fail(LUMO_EINVAL, "%s: act %d (0 or 1)", fn, act);
    if (max_path < 1 || max_path > 4096) return fail(LUMO_EINVAL, "%s: max_path %d (1..4096)", fn, max_path);
    if (dims->n_req == 0) return LUMO_OK;
    LUMO_TRY(check_ptr(state, fn, "state"));
    LUMO_TRY(check_ptr(conv_hist, fn, "conv_hist"));
    LUMO_TRY(check_ptr(w, fn, "w"));
    LUMO_TRY(check_ptr(bias, fn, "bias", true));
    LUMO_TRY(check_ptr(path_out, fn, "path_out"));
    LUMO_TRY(check_ptr(path_len, fn, "path_len"));
    if (pend_desc->plan.total_nodes > 0) {
        LUMO_TRY(check_ptr(x_prev, fn, "x_prev"));
        LUMO_TRY(check_ptr(pend_g, fn, "pend_g"));
        LUMO_TRY(check_ptr(pend_beta, fn, "pend_beta"));
    }
    if (desc->plan.total_nodes > 0) {
        LUMO_TRY(check_ptr(x, fn, "x"));
        LUMO_TRY(check_ptr(g, fn, "g"));
        LUMO_TRY(check_ptr(beta, fn, "beta"));
        LUMO_TRY(check_ptr(o, fn, "o"));
    }
    GdnArgs a{nullptr, nullptr, nullptr, g, beta, state, o, nullptr, nullptr, pr};
    PendArgs pa{pend_desc, max_path, path_out, path_len, nullptr, nullptr, pend_g, pend_beta, state};
    ConvFuseArgs cf{channels, x, conv_hist, w, bias, act, x_prev};
    hipError_t e = launch_wy_conv(*dims, *desc, a, static_cast<hipStream_t>(stream), pa, cf);
    if (e == hipErrorNotSupported) return fail(LUMO_EUNSUPPORTED, "%s: not available for this shape", fn);
    if (e != hipSuccess) return fail(LUMO_EHIP, "%s: launch failed: %s", fn, hipGetErrorString(e));
    return LUMO_OK;
}

namespace {

lumo_status check_commit(const lumo_gdn_dims* dims, const lumo_tree_desc* desc, int32_t max_path,
                         const int32_t* accepted, int32_t* path_out, int32_t* path_len, const void* k,
                         const void* v, const float* g, const float* beta, float* state, int32_t channels,
                         const void* x, void* conv_hist, const char* fn) {
    LUMO_TRY(check_dims(dims, fn));
    LUMO_TRY(check_desc(dims, desc, fn));
    if (max_path < 1 || max_path > 4096) return fail(LUMO_EINVAL, "%s: max_path %d (1..4096)", fn, max_path);
    if (dims->n_req == 0) return LUMO_OK;
    LUMO_TRY(check_ptr(accepted, fn, "accepted_node"));
    LUMO_TRY(check_ptr(path_out, fn, "path_out"));
    LUMO_TRY(check_ptr(path_len, fn, "path_len"));
    LUMO_TRY(check_ptr(state, fn, "state", true));
    if (state) {  // a NULL state defers the replay: the operands are not read
        LUMO_TRY(check_ptr(k, fn, "k"));
        LUMO_TRY(check_ptr(v, fn, "v"));
        LUMO_TRY(check_ptr(g, fn, "g"));
        LUMO_TRY(check_ptr(beta, fn, "beta"));
    }
    if ((x == nullptr) != (conv_hist == nullptr))
        return fail(LUMO_EINVAL, "%s: x and conv_hist must both be given or both be NULL", fn);
    if (x) {
        LUMO_TRY(check_ptr(x, fn, "x"));
        LUMO_TRY(check_ptr(conv_hist, fn, "conv_hist"));
        if (channels <= 0 || channels % 8)
            return fail(LUMO_ESHAPE, "%s: channels %d must be a positive multiple of 8", fn, channels);
    }
    return LUMO_OK;
}

}  // namespace

extern "C" lumo_status lumo_gdn_commit(const lumo_gdn_dims* dims, const lumo_tree_desc* desc, int32_t max_path,
                                       const int32_t* accepted_node, int32_t* path_out, int32_t* path_len,
                                       const void* k, const void* v, const float* g, const float* beta, float* state,
                                       int32_t channels, const void* x, void* conv_hist, void* stream) {
    static const char* fn = "lumo_gdn_commit";
    clear_error();
    LUMO_TRY(check_commit(dims, desc, max_path, accepted_node, path_out, path_len, k, v, g, beta, state, channels, x,
                          conv_hist, fn));
    if (dims->n_req == 0) return LUMO_OK;
    CommitArgs a{max_path, accepted_node, path_out, path_len, k, v, g, beta, state, channels, x, conv_hist};
    hipError_t e = launch_commit(*dims, *desc, a, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return fail(LUMO_EHIP, "%s: launch failed: %s", fn, hipGetErrorString(e));
    return LUMO_OK;
}

extern "C" lumo_status lumo_gdn_commit_prep(const lumo_gdn_dims* dims, const lumo_tree_desc* desc,
                                            const lumo_gdn_prep* prep, int32_t max_path,
                                            const int32_t* accepted_node, int32_t* path_out, int32_t* path_len,
                                            const void* k, const void* v, const float* g, const float* beta,
                                            float* state, int32_t channels, const void* x, void* conv_hist,
                                            void* stream) {
    static const char* fn = "lumo_gdn_commit_prep";
    clear_error();
    LUMO_TRY(check_commit(dims, desc, max_path, accepted_node, path_out, path_len, k, v, g, beta, state, channels, x,
                          conv_hist, fn));
    PrepArgs pr;
    LUMO_TRY(check_prep(prep, fn, pr));
    if (dims->n_req == 0) return LUMO_OK;
    CommitArgs a{max_path, accepted_node, path_out, path_len, k, v, g, beta, state, channels, x, conv_hist, pr};
    hipError_t e = launch_commit(*dims, *desc, a, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return fail(LUMO_EHIP, "%s: launch failed: %s", fn, hipGetErrorString(e));
    return LUMO_OK;
}

extern "C" lumo_status lumo_gdn_commit_hist_layers(const lumo_gdn_dims* dims, const lumo_tree_desc* desc,
                                                   int32_t max_path, const int32_t* accepted_node,
                                                   int32_t* path_out, int32_t* path_len, int32_t channels,
                                                   const void* const* x_layers, void* const* conv_hist_layers,
                                                   void* stream) {
    static const char* fn = "lumo_gdn_commit_hist_layers";
    clear_error();
    LUMO_TRY(check_dims(dims, fn));
    LUMO_TRY(check_desc(dims, desc, fn));
    if (max_path < 1 || max_path > 4096) return fail(LUMO_EINVAL, "%s: max_path %d (1..4096)", fn, max_path);
    if (dims->n_layers > kMaxLayerTable)
        return fail(LUMO_EUNSUPPORTED, "%s: n_layers %d (at most %d)", fn, dims->n_layers, kMaxLayerTable);
    if (channels <= 0 || channels % 8)
        return fail(LUMO_ESHAPE, "%s: channels %d must be a positive multiple of 8", fn, channels);
    if (dims->n_req == 0) return LUMO_OK;
    LUMO_TRY(check_ptr(accepted_node, fn, "accepted_node"));
    LUMO_TRY(check_ptr(path_out, fn, "path_out"));
    LUMO_TRY(check_ptr(path_len, fn, "path_len"));
    if (!x_layers) return fail(LUMO_EINVAL, "%s: x_layers is NULL", fn);
    if (!conv_hist_layers) return fail(LUMO_EINVAL, "%s: conv_hist_layers is NULL", fn);
    for (int l = 0; l < dims->n_layers; ++l) {
        if (desc->plan.total_nodes > 0 && (!x_layers[l] || !aligned16(x_layers[l])))
            return fail(LUMO_EINVAL, "%s: x_layers[%d] is NULL or not 16-byte aligned", fn, l);
        if (!conv_hist_layers[l] || !aligned16(conv_hist_layers[l]))
            return fail(LUMO_EINVAL, "%s: conv_hist_layers[%d] is NULL or not 16-byte aligned", fn, l);
    }
    CommitArgs a{max_path, accepted_node, path_out, path_len, nullptr, nullptr, nullptr, nullptr, nullptr,
                 channels, nullptr, nullptr};
    hipError_t e = launch_commit_hist_layers(*dims, *desc, a, x_layers, conv_hist_layers,
                                             static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return fail(LUMO_EHIP, "%s: launch failed: %s", fn, hipGetErrorString(e));
    return LUMO_OK;
}

namespace {
lumo_status check_attn_dims(const lumo_attn_dims* d, const char* fn) {
    if (!d) return fail(LUMO_EINVAL, "%s: dims is NULL", fn);
    if (d->n_req < 0 || d->h_q < 1 || d->h_kv < 1) return fail(LUMO_ESHAPE, "%s: need n_req >= 0, h_q, h_kv >= 1", fn);
    if (d->h_q % d->h_kv) return fail(LUMO_ESHAPE, "%s: h_q (%d) is not a multiple of h_kv (%d)", fn, d->h_q, d->h_kv);
    const int grp = d->h_q / d->h_kv;
    if (grp != 1 && grp != 2 && grp != 4 && grp != 8)
        return fail(LUMO_EUNSUPPORTED, "%s: h_q / h_kv = %d (supported: 1, 2, 4, 8)", fn, grp);
    if (d->d != 128 || d->op_dtype != LUMO_BF16)
        return fail(LUMO_EUNSUPPORTED, "%s: built for bf16 with d = 128 (got d = %d, dtype %d)", fn, d->d, d->op_dtype);
    return LUMO_OK;
}
}  // namespace

extern "C" size_t lumo_tree_attention_workspace_bytes(const lumo_attn_dims* d, const lumo_plan* p, int32_t n_split) {
    if (!d || !p || n_split < 1) return 0;
    return (size_t)(n_split + 1) * p->total_rows * d->h_q * (128 + 1) * sizeof(float);
}

extern "C" int32_t lumo_tree_attention_splits(const lumo_attn_dims* d, const lumo_plan* p, int32_t max_ctx) {
    if (!d || !p || d->h_kv < 1 || d->h_q < d->h_kv) return 1;
    // Blocks of one partition: requests x kv heads x head blocks x query chunks; the
    // device holds 512 such blocks at once (256 with 4 query heads per block). Pick the
    // partition count that minimises (rounds of resident blocks) x (64-key tiles per
    // block), the longest chain of tiles any block slot runs.
    const int grp = d->h_q / d->h_kv;
    const long per = (long)d->n_req * d->h_kv * (grp > 4 ? grp / 4 : 1) * ((p->max_nodes + 31) / 32);
    const long slots = grp >= 4 ? 256 : 512;
    if (per <= 0 || max_ctx <= 0) return 1;
    const long max_n = std::min<long>(4096, std::max<long>(1, (max_ctx + 63) / 64));
    long best = 1, best_cost = -1;
    for (long n = 1; n <= max_n; ++n) {
        const long rounds = ((n + 1) * per + slots - 1) / slots;
        const long tiles = ((long)attn_part_len(max_ctx, (int)n) + 63) / 64;
        const long cost = rounds * tiles;
        if (best_cost < 0 || cost < best_cost) {
            best = n;
            best_cost = cost;
        }
    }
    return (int32_t)best;
}

extern "C" lumo_status lumo_tree_attention(const lumo_attn_dims* dims, const lumo_tree_desc* desc,
                                           const int32_t* ctx_off, int32_t max_ctx, float scale, const void* q,
                                           const void* k_ctx, const void* v_ctx, const void* k_tree,
                                           const void* v_tree, void* o, float* lse, int32_t n_split,
                                           void* workspace, size_t workspace_bytes, void* stream) {
    static const char* fn = "lumo_tree_attention";
    clear_error();
    LUMO_TRY(check_attn_dims(dims, fn));
    if (!desc) return fail(LUMO_EINVAL, "%s: desc is NULL", fn);
    const lumo_plan& pl = desc->plan;
    if (pl.n_req != dims->n_req) return fail(LUMO_EDESC, "%s: plan has %d requests, dims %d", fn, pl.n_req, dims->n_req);
    if (!desc->blob) return fail(LUMO_EINVAL, "%s: desc blob is NULL", fn);
    if (n_split < 1 || n_split > 4096) return fail(LUMO_EINVAL, "%s: n_split %d (1..4096)", fn, n_split);
    if (max_ctx < 0) return fail(LUMO_EINVAL, "%s: max_ctx %d", fn, max_ctx);
    if (!(scale > 0.f && scale < 3.0e38f)) return fail(LUMO_EINVAL, "%s: scale must be positive and finite", fn);
    if (dims->n_req == 0 || pl.total_nodes == 0) return LUMO_OK;
    LUMO_TRY(check_ptr(ctx_off, fn, "ctx_off"));
    LUMO_TRY(check_ptr(q, fn, "q"));
    LUMO_TRY(check_ptr(k_tree, fn, "k_tree"));
    LUMO_TRY(check_ptr(v_tree, fn, "v_tree"));
    LUMO_TRY(check_ptr(o, fn, "o"));
    LUMO_TRY(check_ptr(lse, fn, "lse"));
    if (max_ctx > 0) {
        LUMO_TRY(check_ptr(k_ctx, fn, "k_ctx"));
        LUMO_TRY(check_ptr(v_ctx, fn, "v_ctx"));
    } else {
        k_ctx = k_tree;  // never read: every context range is empty
        v_ctx = v_tree;
    }
    const size_t need = lumo_tree_attention_workspace_bytes(dims, &pl, n_split);
    LUMO_TRY(check_ptr(workspace, fn, "workspace"));
    if (workspace_bytes < need) return fail(LUMO_ESPACE, "%s: workspace needs %zu bytes, got %zu", fn, need, workspace_bytes);
    AttnArgs a{ctx_off, max_ctx, n_split, scale, q, k_ctx, v_ctx, k_tree, v_tree, o, lse, static_cast<float*>(workspace)};
    hipError_t e = launch_attention(*dims, *desc, a, static_cast<hipStream_t>(stream));
    if (e == hipErrorNotSupported) return fail(LUMO_EUNSUPPORTED, "%s: not compiled into the library", fn);
    if (e != hipSuccess) return fail(LUMO_EHIP, "%s: launch failed: %s", fn, hipGetErrorString(e));
    return LUMO_OK;
}

extern "C" lumo_status lumo_tree_attention_noalloc(const lumo_attn_dims* dims, const lumo_tree_desc* desc,
                                                   const int32_t* ctx_off, int32_t max_ctx, float scale,
                                                   const void* q, const void* k_ctx, const void* v_ctx,
                                                   const void* k_tree, const void* v_tree, void* o, float* lse,
                                                   int32_t n_split, void* stream) {
    static const char* fn = "lumo_tree_attention_noalloc";
    clear_error();
    LUMO_TRY(check_attn_dims(dims, fn));
    if (!desc) return fail(LUMO_EINVAL, "%s: desc is NULL", fn);
    const lumo_plan& pl = desc->plan;
    if (pl.n_req != dims->n_req) return fail(LUMO_EDESC, "%s: plan has %d requests, dims %d", fn, pl.n_req, dims->n_req);
    if (!desc->blob) return fail(LUMO_EINVAL, "%s: desc blob is NULL", fn);
    if (n_split < 1 || n_split > 4096) return fail(LUMO_EINVAL, "%s: n_split %d (1..4096)", fn, n_split);
    if (max_ctx < 0) return fail(LUMO_EINVAL, "%s: max_ctx %d", fn, max_ctx);
    if (!(scale > 0.f && scale < 3.0e38f)) return fail(LUMO_EINVAL, "%s: scale must be positive and finite", fn);
    const size_t need = lumo_tree_attention_workspace_bytes(dims, &pl, n_split);
    if (need > (size_t)LUMO_TREE_ATTENTION_SCRATCH_BYTES)
        return fail(LUMO_ESPACE,
                    "%s: the partial results need %zu bytes, more than the fixed %u-byte scratch array; "
                    "use fewer splits (n_split %d) or lumo_tree_attention with a workspace",
                    fn, need, (unsigned)LUMO_TREE_ATTENTION_SCRATCH_BYTES, n_split);
    if (dims->n_req == 0 || pl.total_nodes == 0) return LUMO_OK;
    LUMO_TRY(check_ptr(ctx_off, fn, "ctx_off"));
    LUMO_TRY(check_ptr(q, fn, "q"));
    LUMO_TRY(check_ptr(k_tree, fn, "k_tree"));
    LUMO_TRY(check_ptr(v_tree, fn, "v_tree"));
    LUMO_TRY(check_ptr(o, fn, "o"));
    LUMO_TRY(check_ptr(lse, fn, "lse"));
    if (max_ctx > 0) {
        LUMO_TRY(check_ptr(k_ctx, fn, "k_ctx"));
        LUMO_TRY(check_ptr(v_ctx, fn, "v_ctx"));
    } else {
        k_ctx = k_tree;  // never read: every context range is empty
        v_ctx = v_tree;
    }
    float* ws = nullptr;
    hipError_t e = attn_scratch(&ws);
    if (e != hipSuccess) return fail(LUMO_EHIP, "%s: scratch address lookup failed: %s", fn, hipGetErrorString(e));
    AttnArgs a{ctx_off, max_ctx, n_split, scale, q, k_ctx, v_ctx, k_tree, v_tree, o, lse, ws};
    e = launch_attention(*dims, *desc, a, static_cast<hipStream_t>(stream));
    if (e == hipErrorNotSupported) return fail(LUMO_EUNSUPPORTED, "%s: not compiled into the library", fn);
    if (e != hipSuccess) return fail(LUMO_EHIP, "%s: launch failed: %s", fn, hipGetErrorString(e));
    return LUMO_OK;
}

extern "C" size_t lumo_draft_select_workspace_bytes(int32_t rows, int32_t k, int32_t n_split) {
    if (rows < 0 || k < 1 || n_split <= 1) return 0;
    return (size_t)rows * n_split * 4 * (k + 1) * sizeof(uint64_t);  // one entry per wavefront
}

extern "C" int32_t lumo_draft_select_splits(int32_t rows, int32_t vocab, int32_t dtype) {
    // Parts of at least 2048 16-byte vectors (eight per thread, one batch) and at most
    // 1024 blocks in all: the best measured points for 1, 8 and 64 rows of 248,320
    // logits lie there.
    if (rows < 1 || vocab < 1) return 1;
    const long per_vec = dtype == LUMO_BF16 ? 8 : 4;
    const long nvec = (long)vocab / per_vec;
    const long want = nvec / 2048;
    const long cap = std::max<long>(1, 1024 / rows);
    return (int32_t)std::max<long>(1, std::min<long>({want, cap, 4096}));
}

extern "C" lumo_status lumo_draft_select(int32_t rows, int32_t vocab, int64_t ld, int32_t dtype, int32_t k,
                                         int32_t ties, const void* logits, int32_t* spine, int32_t* cand,
                                         int32_t n_split, void* workspace, size_t workspace_bytes, void* stream) {
    static const char* fn = "lumo_draft_select";
    clear_error();
    if (rows < 0) return fail(LUMO_EINVAL, "%s: rows %d", fn, rows);
    if (vocab < 1) return fail(LUMO_EINVAL, "%s: vocab %d", fn, vocab);
    if (ld < vocab) return fail(LUMO_EINVAL, "%s: ld %lld < vocab %d", fn, (long long)ld, vocab);
    if (dtype != LUMO_F32 && dtype != LUMO_BF16) return fail(LUMO_EUNSUPPORTED, "%s: dtype %d", fn, dtype);
    if (ties != 0 && ties != 1) return fail(LUMO_EINVAL, "%s: ties %d (0 or 1)", fn, ties);
    if (k < 1 || k > vocab) return fail(LUMO_EINVAL, "%s: k %d (1..vocab %d)", fn, k, vocab);
    if (k > 8) return fail(LUMO_EUNSUPPORTED, "%s: k %d (at most 8)", fn, k);
    if (n_split < 1 || n_split > 4096) return fail(LUMO_EINVAL, "%s: n_split %d (1..4096)", fn, n_split);
    // element offsets and the grid stay within their index types
    if ((long long)rows * n_split > 0x7fffffffLL) return fail(LUMO_EINVAL, "%s: rows x n_split too large", fn);
    if (rows > 0 && (ld > (1LL << 40) || (long long)(rows - 1) * ld + vocab > (1LL << 40)))
        return fail(LUMO_EINVAL, "%s: logits span too large", fn);
    if (rows == 0) return LUMO_OK;
    LUMO_TRY(check_ptr(logits, fn, "logits"));
    LUMO_TRY(check_ptr(spine, fn, "spine"));
    LUMO_TRY(check_ptr(cand, fn, "cand"));
    uint64_t* parts = nullptr;
    if (n_split > 1) {
        const size_t need = lumo_draft_select_workspace_bytes(rows, k, n_split);
        LUMO_TRY(check_ptr(workspace, fn, "workspace"));
        if (workspace_bytes < need)
            return fail(LUMO_ESPACE, "%s: workspace needs %zu bytes, got %zu", fn, need, workspace_bytes);
        parts = static_cast<uint64_t*>(workspace);
    }
    SelectArgs a{logits, rows, vocab, (long)ld, dtype, k, ties, n_split, spine, cand, parts};
    hipError_t e = launch_select(a, static_cast<hipStream_t>(stream));
    if (e == hipErrorNotSupported) return fail(LUMO_EUNSUPPORTED, "%s: not compiled into the library", fn);
    if (e != hipSuccess) return fail(LUMO_EHIP, "%s: launch failed: %s", fn, hipGetErrorString(e));
    return LUMO_OK;
}

struct lumo_commit_graph {
    hipGraph_t graph = nullptr;
    hipGraphExec_t exec = nullptr;
};

extern "C" lumo_status lumo_gdn_commit_graph_create(const lumo_gdn_dims* dims, const lumo_tree_desc* desc,
                                                    const lumo_gdn_prep* prep, int32_t max_path,
                                                    const int32_t* accepted_node, int32_t* path_out,
                                                    int32_t* path_len, const void* k, const void* v, const float* g,
                                                    const float* beta, float* state, int32_t channels, const void* x,
                                                    void* conv_hist, lumo_commit_graph** out) {
    static const char* fn = "lumo_gdn_commit_graph_create";
    clear_error();
    if (!out) return fail(LUMO_EINVAL, "%s: out is NULL", fn);
    *out = nullptr;
    LUMO_TRY(check_commit(dims, desc, max_path, accepted_node, path_out, path_len, k, v, g, beta, state, channels, x,
                          conv_hist, fn));
    PrepArgs pr;
    LUMO_TRY(check_prep(prep, fn, pr));
    lumo_commit_graph* cg = new (std::nothrow) lumo_commit_graph();
    if (!cg) return fail(LUMO_EHIP, "%s: out of host memory", fn);
    hipStream_t s = nullptr;
    hipError_t e = hipStreamCreateWithFlags(&s, hipStreamNonBlocking);
    if (e == hipSuccess) e = hipStreamBeginCapture(s, hipStreamCaptureModeThreadLocal);
    if (e == hipSuccess) {
        hipError_t le = hipSuccess;
        if (dims->n_req > 0) {
            CommitArgs a{max_path, accepted_node, path_out, path_len, k, v, g, beta, state, channels, x, conv_hist, pr};
            le = launch_commit(*dims, *desc, a, s);
        }
        e = hipStreamEndCapture(s, &cg->graph);
        if (e == hipSuccess) e = le;
    }
    if (e == hipSuccess) e = hipGraphInstantiate(&cg->exec, cg->graph, nullptr, nullptr, 0);
    if (s) (void)hipStreamDestroy(s);
    if (e != hipSuccess) {
        if (cg->exec) (void)hipGraphExecDestroy(cg->exec);
        if (cg->graph) (void)hipGraphDestroy(cg->graph);
        delete cg;
        return fail(LUMO_EHIP, "%s: capture failed: %s", fn, hipGetErrorString(e));
    }
    *out = cg;
    return LUMO_OK;
}

extern "C" lumo_status lumo_gdn_commit_graph_launch(lumo_commit_graph* graph, void* stream) {
    clear_error();
    if (!graph || !graph->exec) return fail(LUMO_EINVAL, "lumo_gdn_commit_graph_launch: graph is NULL");
    hipError_t e = hipGraphLaunch(graph->exec, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return fail(LUMO_EHIP, "lumo_gdn_commit_graph_launch: %s", hipGetErrorString(e));
    return LUMO_OK;
}

extern "C" void lumo_gdn_commit_graph_destroy(lumo_commit_graph* graph) {
    if (!graph) return;
    if (graph->exec) (void)hipGraphExecDestroy(graph->exec);
    if (graph->graph) (void)hipGraphDestroy(graph->graph);
    delete graph;
}
