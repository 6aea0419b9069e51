// Tree causal convolution (LumoTree Sec. V-C, Tab. II row 3).
//
// The planner turns the topology into static gather sources: for every node, the
// four rows of its window (oldest first), each either an x row along the ancestry
// or a committed-history entry. The kernel gathers those rows and applies the four
// taps in order with fp32 accumulation starting from the bias, then the activation,
// then one cast. One thread handles 8 contiguous channels of one layer for a run of
// nodes; loads and stores are 16-byte vectors, the thread's taps stay in registers,
// and every x row is read by at most four nodes (itself and three descendants, which
// follow it closely in node order, so the re-reads hit L2). HBM-bound.
#include "device_common.h"
#include "internal.h"
#include "launch.h"

namespace lumo {
namespace {

struct ConvParams {
    const int32_t* blob;
    int32_t o_req, o_row, o_conv_src;
    int32_t total_nodes, total_rows, n_layers, channels, n_cchunks, act;
    const void* x;
    const void* hist;
    const float* w;
    const float* bias;
    void* y;
};

template <int OPT> struct Vec8;
template <> struct Vec8<0> {
    struct Raw {
        float4 a, b;
    };
    static __device__ __forceinline__ Raw ld_raw(const float* p) {
        return Raw{reinterpret_cast<const float4*>(p)[0], reinterpret_cast<const float4*>(p)[1]};
    }
    static __device__ __forceinline__ void unpack(const Raw& w, float (&v)[8]) {
        v[0] = w.a.x; v[1] = w.a.y; v[2] = w.a.z; v[3] = w.a.w;
        v[4] = w.b.x; v[5] = w.b.y; v[6] = w.b.z; v[7] = w.b.w;
    }
    static __device__ __forceinline__ void st(float* p, const float (&v)[8]) {
        reinterpret_cast<float4*>(p)[0] = make_float4(v[0], v[1], v[2], v[3]);
        reinterpret_cast<float4*>(p)[1] = make_float4(v[4], v[5], v[6], v[7]);
    }
};
template <> struct Vec8<1> {
    using Raw = uint4;
    static __device__ __forceinline__ Raw ld_raw(const uint16_t* p) { return reinterpret_cast<const uint4*>(p)[0]; }
    static __device__ __forceinline__ void unpack(const Raw& a, float (&v)[8]) {
        v[0] = bf16_lo(a.x); v[1] = bf16_hi(a.x); v[2] = bf16_lo(a.y); v[3] = bf16_hi(a.y);
        v[4] = bf16_lo(a.z); v[5] = bf16_hi(a.z); v[6] = bf16_lo(a.w); v[7] = bf16_hi(a.w);
    }
    static __device__ __forceinline__ void st(uint16_t* p, const float (&v)[8]) {
        uint4 a;
        a.x = f32x2_to_bf16x2(v[0], v[1]);
        a.y = f32x2_to_bf16x2(v[2], v[3]);
        a.z = f32x2_to_bf16x2(v[4], v[5]);
        a.w = f32x2_to_bf16x2(v[6], v[7]);
        reinterpret_cast<uint4*>(p)[0] = a;
    }
};

// One block: one layer, 2048 channels (8 per thread), a run of kNodesPerBlock nodes.
// The taps and bias of the thread's channels stay in registers across the run; the
// window rows of consecutive nodes (parents, grandparents) are mostly L2 hits.
constexpr int kNodesPerBlock = 32;

template <int OPT>
__global__ __launch_bounds__(256) void conv_kernel(ConvParams p) {
    using T = typename Op<OPT>::T;
    int t = xcd_remap(blockIdx.x, gridDim.x);
    const int ng = (p.total_nodes + kNodesPerBlock - 1) / kNodesPerBlock;
    const int grp = t % ng;
    t /= ng;
    const int cc = t % p.n_cchunks;
    const int l = t / p.n_cchunks;
    // channel-less threads stay alive: their lanes still carry node info for readlane
    const int c0ch = (cc * 256 + (int)threadIdx.x) * 8;
    const bool has_c = c0ch < p.channels;
    const int c = has_c ? c0ch : p.channels - 8;
    const T* x = static_cast<const T*>(p.x);
    const T* hist = static_cast<const T*>(p.hist);
    T* y = static_cast<T*>(p.y);
    float wt[32];
    const float4* wp = reinterpret_cast<const float4*>(p.w + ((long)l * p.channels + c) * 4);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const float4 q = wp[e];
        wt[4 * e] = q.x; wt[4 * e + 1] = q.y; wt[4 * e + 2] = q.z; wt[4 * e + 3] = q.w;
    }
    float b0[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) b0[e] = p.bias ? p.bias[(long)l * p.channels + c + e] : 0.f;
    const int n0 = grp * kNodesPerBlock;
    const int nn = min(p.total_nodes, n0 + kNodesPerBlock) - n0;
    // node info of the run, one node per lane (lanes 0..31 of every wave), broadcast
    // per node with readlane so the window loads depend on nothing but registers
    const int li = (int)threadIdx.x & (kNodesPerBlock - 1);
    const int mine = n0 + (li < nn ? li : 0);
    const int i_req = p.blob[p.o_req + mine];
    const int i_row = p.blob[p.o_row + mine];
    int i_src[4];
#pragma unroll
    for (int tap = 0; tap < 4; ++tap) i_src[tap] = p.blob[p.o_conv_src + 4 * mine + tap];
    // kBatch nodes per step: all their window loads are issued before any is used
    constexpr int kBatch = 4;
    for (int i0 = 0; i0 < nn; i0 += kBatch) {
        typename Vec8<OPT>::Raw raw[kBatch][4];
#pragma unroll
        for (int bi = 0; bi < kBatch; ++bi) {
            const int i = min(i0 + bi, nn - 1);  // past the run: reload the last node, not stored
            const int r = __builtin_amdgcn_readlane(i_req, i);
#pragma unroll
            for (int tap = 0; tap < 4; ++tap) {
                const int s = __builtin_amdgcn_readlane(i_src[tap], i);
                const T* rp = s >= 0 ? x + ((long)l * p.total_rows + s) * p.channels + c
                                     : hist + (((long)r * p.n_layers + l) * 3 + (-1 - s)) * p.channels + c;
                raw[bi][tap] = Vec8<OPT>::ld_raw(rp);
            }
        }
#pragma unroll
        for (int bi = 0; bi < kBatch; ++bi) {
            if (i0 + bi >= nn) break;
            const int row = __builtin_amdgcn_readlane(i_row, i0 + bi);
            float acc[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[e] = b0[e];
#pragma unroll
            for (int tap = 0; tap < 4; ++tap) {
                float xv[8];
                Vec8<OPT>::unpack(raw[bi][tap], xv);
#pragma unroll
                for (int e = 0; e < 8; ++e) acc[e] = __builtin_fmaf(wt[4 * e + tap], xv[e], acc[e]);
            }
            if (p.act == 1) {  // SiLU: x sigmoid(x), with the hardware reciprocal (<= 1 ulp)
#pragma unroll
                for (int e = 0; e < 8; ++e) acc[e] = acc[e] * __builtin_amdgcn_rcpf(1.f + __expf(-acc[e]));
            }
            if (has_c) Vec8<OPT>::st(y + ((long)l * p.total_rows + row) * p.channels + c, acc);
        }
    }
}

}  // namespace

hipError_t launch_conv(const lumo_gdn_dims& d, const lumo_tree_desc& desc, const ConvArgs& a, hipStream_t s) {
    const lumo_plan& pl = desc.plan;
    if (pl.total_nodes == 0) return hipSuccess;
    ConvParams p;
    p.blob = desc.blob;
    p.o_req = pl.o_req;
    p.o_row = pl.o_row;
    p.o_conv_src = pl.o_conv_src;
    p.total_nodes = pl.total_nodes;
    p.total_rows = pl.total_rows;
    p.n_layers = d.n_layers;
    p.channels = a.channels;
    p.n_cchunks = (a.channels + 2047) / 2048;
    p.act = a.act;
    p.x = a.x;
    p.hist = a.hist;
    p.w = a.w;
    p.bias = a.bias;
    p.y = a.y;
    const long blocks = (long)d.n_layers * p.n_cchunks * ((pl.total_nodes + kNodesPerBlock - 1) / kNodesPerBlock);
    if (d.op_dtype == LUMO_BF16)
        hipLaunchKernelGGL(conv_kernel<1>, dim3((unsigned)blocks), dim3(256), 0, s, p);
    else
        hipLaunchKernelGGL(conv_kernel<0>, dim3((unsigned)blocks), dim3(256), 0, s, p);
    return hipGetLastError();
}

}  // namespace lumo
