// Host launchers of the gfx950 kernels (arguments already validated by the C ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "lumo_tree.h"

namespace lumo {

// Operand preparation inside the kernels (lumo_gdn_prep); flags 0 = operands as given.
struct PrepArgs {
    int32_t flags = 0;
    float qk_eps = 0.f;
    const float* a_log = nullptr;
    const float* dt_bias = nullptr;
};

struct GdnArgs {
    const void* q;
    const void* k;
    const void* v;
    const float* g;
    const float* beta;
    const float* state0;
    void* o;
    float* node_states;
    float* ws;
    PrepArgs prep;  // WY kernel, and the scans of lumo_tree_gdn_verify_prep
};

// Sequential path scans (PATHS / TWO_LEVEL / RECOMPUTE): one launch per dependency level.
hipError_t launch_scan(const lumo_gdn_dims& d, const lumo_tree_desc& desc, const GdnArgs& a, hipStream_t s);

// A pending accepted path of the previous iteration, replayed into the state bank by
// the WY kernel before it verifies (lumo_tree_gdn_verify_pending).
struct PendArgs {
    const lumo_tree_desc* desc;  // previous iteration's descriptor
    int32_t max_path;
    const int32_t* path_out;
    const int32_t* path_len;
    const void* k;
    const void* v;
    const float* g;
    const float* beta;
    float* state;  // in/out; the verification reads the published state from here
};

// Tree WY form on MFMA: one launch, no workspace. With `pend`, the pending path is
// published into pend->state first (a.state0 is ignored) and requests without nodes
// in `desc` are still published.
hipError_t launch_wy(const lumo_gdn_dims& d, const lumo_tree_desc& desc, const GdnArgs& a, hipStream_t s,
                     const PendArgs* pend = nullptr);

// The tree conv fused into the WY verification: q, k and v are the conv outputs of x
// (channels q | k | v), computed in the kernel and never stored; the history is
// published from the pending path (when one is pending) and read from hist. With this,
// GdnArgs q, k, v and PendArgs k, v are unused.
struct ConvFuseArgs {
    int32_t channels;
    const void* x;        // [layers][rows][channels]
    void* hist;           // [req][layers][3][channels], published in place
    const float* w;       // [layers][channels][4]
    const float* bias;    // [layers][channels] or NULL
    int32_t act;
    const void* x_prev;   // the pending path's x rows: [layers][previous rows][channels]
};
hipError_t launch_wy_conv(const lumo_gdn_dims& d, const lumo_tree_desc& desc, const GdnArgs& a, hipStream_t s,
                          const PendArgs& pend, const ConvFuseArgs& cf);
constexpr int kWyMaxDepth = 17;  // nodes on a root-to-leaf path

// The WY form on the vector ALUs for the shapes the matrix-core kernel does not take
// (fp32 operands, d_k or d_v below 128, paths of 18 to kWyvMaxDepth nodes). No
// workspace; operand preparation as in GdnArgs::prep.
constexpr int kWyvMaxDepth = 32;
hipError_t launch_wyv(const lumo_gdn_dims& d, const lumo_tree_desc& desc, const GdnArgs& a, hipStream_t s);
// Whether the matrix-core WY kernel serves these dimensions and plan.
inline bool wy_mfma_shape(const lumo_gdn_dims& d, const lumo_plan& p) {
    return d.op_dtype == LUMO_BF16 && d.d_k == 128 && d.d_v == 128 && p.max_depth <= kWyMaxDepth;
}

struct CommitArgs {
    int32_t max_path;
    const int32_t* accepted;
    int32_t* path_out;
    int32_t* path_len;
    const void* k;
    const void* v;
    const float* g;
    const float* beta;
    float* state;
    int32_t channels;
    const void* x;
    void* conv_hist;
    PrepArgs prep;  // replay only
};

hipError_t launch_commit(const lumo_gdn_dims& d, const lumo_tree_desc& desc, const CommitArgs& a, hipStream_t s);

struct ConvArgs {
    int32_t channels;
    const void* x;
    const void* hist;
    const float* w;
    const float* bias;
    int32_t act;
    void* y;
};

// The previous iteration's accepted path, published into the conv history by the conv
// of this iteration (lumo_tree_conv_gather_pending).
struct ConvPendArgs {
    const lumo_tree_desc* desc;  // previous iteration's descriptor
    int32_t max_path;
    const int32_t* path_out;
    const int32_t* path_len;
    const void* x_prev;
};

hipError_t launch_conv(const lumo_gdn_dims& d, const lumo_tree_desc& desc, const ConvArgs& a, hipStream_t s,
                       const ConvPendArgs* pend = nullptr);

// Tree attention: split-K partial kernel plus the merge (workspace: n_split + 1 ranges).
struct AttnArgs {
    const int32_t* ctx_off;
    int32_t max_ctx;
    int32_t n_split;
    float scale;
    const void* q;
    const void* k_ctx;
    const void* v_ctx;
    const void* k_tree;
    const void* v_tree;
    void* o;
    float* lse;
    float* ws;
};
int attn_part_len(int max_ctx, int n_split);
hipError_t launch_attention(const lumo_attn_dims& d, const lumo_tree_desc& desc, const AttnArgs& a, hipStream_t s);
// Device address of the current device's fixed attention scratch array
// (LUMO_TREE_ATTENTION_SCRATCH_BYTES), looked up once per device.
hipError_t attn_scratch(float** out);

}  // namespace lumo
