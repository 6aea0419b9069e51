// Path-parallel tree verification by sequential path scans (LumoTree Sec. IV-A,
// Alg. 2; Eq. (2)-(3)).
//
// One wavefront per (segment, layer, value head, 64-wide value tile). Each lane owns
// one value row j of the head matrix R (the full key dimension, d_k fp32 values, in
// VGPRs) and carries it through every node of its segment: the state tile is loaded
// once (pre-tree state or an exported cut state) and reused across the path loop.
// Rows of R evolve independently, so the k.R and R.q contractions are lane-local;
// the node's k and q rows are wave-uniform and are read with scalar loads.
// Segments of a dependency level are independent and run in one launch; a segment
// exports its tile to the workspace at nodes whose other children start segments of
// the next level (cut states, Sec. IV-C, Eq. (4)). With operand preparation (Sec.
// IV-B) the gates come from raw inputs and the key and query rows are used divided by
// sqrt(|x|^2 + eps), computed as the commit's replay computes them.
#include "device_common.h"
#include "internal.h"
#include "launch.h"

namespace lumo {
namespace {

// Pointers are separate __restrict__ kernel arguments so that the compiler may read
// the wave-uniform key and query rows with scalar loads.
struct ScanParams {
    const int32_t* blob;
    int32_t o_seg, o_seg_nodes;
    int32_t n_layers, total_rows, h_k, h_v, d_v, group, n_vtiles;
    int32_t seg_first;
    PrepArgs prep;  // operand preparation (Sec. IV-B); flags 0 = operands as given
};

template <int DK, int OPT>
__global__ __launch_bounds__(64) void scan_kernel(ScanParams p, const typename Op<OPT>::T* __restrict__ q,
                                                  const typename Op<OPT>::T* __restrict__ k,
                                                  const typename Op<OPT>::T* __restrict__ v,
                                                  const float* __restrict__ g, const float* __restrict__ gbeta,
                                                  const float* __restrict__ state0,
                                                  typename Op<OPT>::T* __restrict__ o,
                                                  float* __restrict__ node_states, float* __restrict__ ws) {
    int t = xcd_remap(blockIdx.x, gridDim.x);
    const int vt = t % p.n_vtiles;
    t /= p.n_vtiles;
    const int h = t % p.h_v;
    t /= p.h_v;
    const int l = t % p.n_layers;
    const int s = p.seg_first + t / p.n_layers;

    const int j = vt * 64 + (int)threadIdx.x;
    const bool act = j < p.d_v;
    const int jc = act ? j : p.d_v - 1;
    const int hk = h / p.group;
    const int32_t* seg = p.blob + p.o_seg + kSegWords * s;
    const int req = seg[0], src = seg[1], first = seg[2], len = seg[3];
    const long mat = (long)DK * p.d_v;

    const float* S0 = src < 0 ? state0 + (((long)req * p.n_layers + l) * p.h_v + h) * mat
                              : ws + (((long)src * p.n_layers + l) * p.h_v + h) * mat;
    float S[DK];
#pragma unroll
    for (int i = 0; i < DK; ++i) S[i] = S0[(long)i * p.d_v + jc];

    const bool qkn = (p.prep.flags & LUMO_PREP_QK_NORM) != 0;  // uniform
    const bool rawg = (p.prep.flags & LUMO_PREP_RAW_GATES) != 0;
    const float alog = rawg ? p.prep.a_log[l * p.h_v + h] : 0.f;
    const float dtb = rawg ? p.prep.dt_bias[l * p.h_v + h] : 0.f;
    for (int e = first; e < first + len; ++e) {
        const int32_t* en = p.blob + p.o_seg_nodes + kSegNodeWords * e;
        const int row = en[0], wout = en[1], cut = en[2];
        const long gi = ((long)l * p.total_rows + row) * p.h_v + h;
        const long ki = (((long)l * p.total_rows + row) * p.h_k + hk) * DK;
        const float gv = g[gi], bv = gbeta[gi];
        const float alpha = __expf(rawg ? raw_log_alpha(gv, alog, dtb) : gv);
        const float beta = rawg ? raw_beta(bv) : bv;
        const float vj = Op<OPT>::ld(v, gi * p.d_v + jc);
        const float ks = qkn ? row_rsq_norm<DK, OPT>(k + ki, p.prep.qk_eps) : 1.f;
        gdn_row_update<DK, OPT>(S, k + ki, vj, alpha, beta, ks);
        if (wout) {
            const float qs = qkn ? row_rsq_norm<DK, OPT>(q + ki, p.prep.qk_eps) : 1.f;
            const float ov = gdn_row_output<DK, OPT>(S, q + ki, qs);
            if (act) {
                Op<OPT>::st(o, gi * p.d_v + j, ov);
                if (node_states) {
                    float* dst = node_states + gi * mat;
#pragma unroll
                    for (int i = 0; i < DK; ++i) dst[(long)i * p.d_v + j] = S[i];
                }
            }
        }
        if (cut >= 0 && act) {
            float* dst = ws + (((long)cut * p.n_layers + l) * p.h_v + h) * mat;
#pragma unroll
            for (int i = 0; i < DK; ++i) dst[(long)i * p.d_v + j] = S[i];
        }
    }
}

template <int DK, int OPT>
void launch_one(dim3 grid, hipStream_t s, const ScanParams& p, const GdnArgs& a) {
    using T = typename Op<OPT>::T;
    hipLaunchKernelGGL((scan_kernel<DK, OPT>), grid, dim3(64), 0, s, p, static_cast<const T*>(a.q),
                       static_cast<const T*>(a.k), static_cast<const T*>(a.v), a.g, a.beta, a.state0,
                       static_cast<T*>(a.o), a.node_states, a.ws);
}

template <int OPT>
hipError_t launch_dk(int dk, dim3 grid, hipStream_t s, const ScanParams& p, const GdnArgs& a) {
    switch (dk) {
        case 16: launch_one<16, OPT>(grid, s, p, a); break;
        case 32: launch_one<32, OPT>(grid, s, p, a); break;
        case 64: launch_one<64, OPT>(grid, s, p, a); break;
        default: launch_one<128, OPT>(grid, s, p, a); break;
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_scan(const lumo_gdn_dims& d, const lumo_tree_desc& desc, const GdnArgs& a, hipStream_t s) {
    const lumo_plan& pl = desc.plan;
    ScanParams p;
    p.blob = desc.blob;
    p.o_seg = pl.o_seg;
    p.o_seg_nodes = pl.o_seg_nodes;
    p.n_layers = d.n_layers;
    p.total_rows = pl.total_rows;
    p.h_k = d.h_k;
    p.h_v = d.h_v;
    p.d_v = d.d_v;
    p.group = d.h_v / d.h_k;
    p.n_vtiles = (d.d_v + 63) / 64;
    p.prep = a.prep;
    // Level boundaries come from the host copy of the plan words.
    for (int lv = 0; lv < pl.n_levels; ++lv) {
        const int first = desc.host_blob[pl.o_level_off + lv];
        const int count = desc.host_blob[pl.o_level_off + lv + 1] - first;
        if (count <= 0) continue;
        p.seg_first = first;
        const long blocks = (long)count * d.n_layers * d.h_v * p.n_vtiles;
        hipError_t e = d.op_dtype == LUMO_BF16 ? launch_dk<1>(d.d_k, dim3((unsigned)blocks), s, p, a)
                                               : launch_dk<0>(d.d_k, dim3((unsigned)blocks), s, p, a);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace lumo
