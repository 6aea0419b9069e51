// Tree causal convolution (LumoTree Sec. V-C, Tab. II row 3).
//
// The planner turns the topology into static gather sources: for every node, the
// four rows of its window (oldest first), each either an x row along the ancestry
// or a committed-history entry. The kernel gathers those rows and applies the four
// taps in order with fp32 accumulation starting from the bias, then the activation,
// then one cast. One thread handles 8 contiguous channels of one layer for a run of
// nodes; loads and stores are 16-byte vectors, the thread's taps stay in registers,
// and every x row is read by at most four nodes (itself and three descendants, which
// follow it closely in each request's depth-first preorder, so most re-reads hit L2).
// HBM-bound.
#include "device_common.h"
#include "internal.h"
#include "launch.h"

namespace lumo {
namespace {

struct ConvParams {
    const int32_t* blob;
    int32_t o_req, o_row, o_conv_src, o_node_off, o_dfs;
    int32_t n_req, total_nodes, total_rows, n_layers, channels, n_cchunks, act;
    int32_t run;  // nodes per block (1..kNodesPerBlock)
    int32_t pre;  // 1: runs follow each request's preorder; 0: the stored node order
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

// Publication of the previous iteration's accepted path into the conv history, deferred
// into this iteration's conv (Alg. 1: iteration t-1's path is published before
// iteration t reads the history). The history of (request r, layer l) becomes the last
// three entries of (history, rows of the previous x along the pending path), in place,
// before the windows read it. A pending length <= 0 or > max_path, or a previous tree
// without nodes, leaves the history as it is.
struct HistPend {
    const int32_t* blob;  // previous iteration's plan
    int32_t o_node_off, o_row, total_rows, max_path;
    const int32_t* path_out;  // [n_req][max_path], root first
    const int32_t* path_len;  // [n_req]
    const void* x_prev;       // previous iteration's x, [layers][its rows][channels]
    void* hist;               // the history, written in place
};

__device__ __forceinline__ int pend_hist_len(const HistPend& q, int r) {
    const int len = q.path_len[r];
    return (len > q.max_path || q.blob[q.o_node_off + r + 1] <= q.blob[q.o_node_off + r]) ? 0 : len;
}

// Source of entry e (0..2) of the published history at channel c, len >= 1: entry
// len + e of (history, previous x rows of the path). Path entries are clamped to the
// previous tree's nodes.
template <class T>
__device__ __forceinline__ const T* pend_hist_src(const HistPend& q, const T* hist_rl, int r, int l, int len,
                                                  int e, int channels, int c) {
    const int pos = len + e;
    if (pos < 3) return hist_rl + (long)pos * channels + c;
    const int base = q.blob[q.o_node_off + r];
    const int pn = q.blob[q.o_node_off + r + 1] - base;
    const int node = min(max(q.path_out[(long)r * q.max_path + pos - 3], 0), pn - 1);
    const int row = q.blob[q.o_row + base + node];
    return static_cast<const T*>(q.x_prev) + ((long)l * q.total_rows + row) * channels + c;
}

// Standalone publication, ahead of the run kernel: one block per (request, layer,
// 2048 channels), 8 channels per thread. The path's first 64 nodes are loaded with its
// length (lane k: entry k), so a published entry's row is one dependent load away.
template <int OPT>
__global__ __launch_bounds__(256) void hist_pend_kernel(HistPend q, int n_layers, int channels, int n_cchunks) {
    using T = typename Op<OPT>::T;
    const int cc = blockIdx.x % n_cchunks;
    const int l = (blockIdx.x / n_cchunks) % n_layers;
    const int r = blockIdx.x / (n_cchunks * n_layers);
    const int pe = q.path_out[(long)r * q.max_path + min((int)threadIdx.x & 63, q.max_path - 1)];
    const int len = pend_hist_len(q, r);
    if (len <= 0) return;  // uniform
    const int c0 = (cc * 256 + (int)threadIdx.x) * 8;
    const bool has_c = c0 < channels;
    const int c = has_c ? c0 : channels - 8;
    T* h = static_cast<T*>(q.hist) + (((long)r * n_layers + l) * 3) * channels;
    const int base = q.blob[q.o_node_off + r];
    const int pn = q.blob[q.o_node_off + r + 1] - base;
    // entry len + e of (history, previous x rows of the path), as pend_hist_src
    auto src = [&](int e) -> const T* {
        const int pos = len + e;  // uniform
        if (pos < 3) return h + (long)pos * channels + c;
        const int k = pos - 3;
        const int nd = k < 64 ? __builtin_amdgcn_readlane(pe, k) : q.path_out[(long)r * q.max_path + k];
        const int row = q.blob[q.o_row + base + min(max(nd, 0), pn - 1)];
        return static_cast<const T*>(q.x_prev) + ((long)l * q.total_rows + row) * channels + c;
    };
    const T* s0 = src(0);
    const T* s1 = src(1);
    const T* s2 = src(2);
    constexpr int W = 16 / sizeof(T) >= 8 ? 1 : 2;  // 16-byte pieces per 8 channels
#pragma unroll
    for (int w = 0; w < W; ++w) {  // each piece read whole before it is overwritten
        const uint4 v0 = reinterpret_cast<const uint4*>(s0)[w];
        const uint4 v1 = reinterpret_cast<const uint4*>(s1)[w];
        const uint4 v2 = reinterpret_cast<const uint4*>(s2)[w];
        if (!has_c) continue;
        reinterpret_cast<uint4*>(h + c)[w] = v0;
        reinterpret_cast<uint4*>(h + (long)channels + c)[w] = v1;
        reinterpret_cast<uint4*>(h + 2L * channels + c)[w] = v2;
    }
}

// One block: one layer, 2048 channels (8 per thread), a run of up to kNodesPerBlock
// nodes (shorter runs when the grid would otherwise leave CUs idle).
// The taps and bias of the thread's channels stay in registers across the run; the
// window rows of nodes close in preorder (parents, grandparents) are mostly L2 hits.
constexpr int kNodesPerBlock = 32;

template <int OPT>
__global__ __launch_bounds__(256) void conv_kernel(ConvParams p) {
    using T = typename Op<OPT>::T;
    int t = xcd_remap(blockIdx.x, gridDim.x);
    const int ng = (p.total_nodes + p.run - 1) / p.run;
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
    const int n0 = grp * p.run;
    const int nn = min(p.total_nodes, n0 + p.run) - n0;
    // node info of the run, one node per lane (lanes 0..31 of every wave), broadcast
    // per node with readlane so the window loads depend on nothing but registers. Full
    // runs cover each request's nodes in depth-first preorder (positions node_off[r] ..),
    // so a node's parent and grandparents were loaded shortly before, by this run or a
    // neighbouring one on the same XCD. Shortened runs (small grids, bound by the
    // latency of their dependent loads) take the nodes in their stored order, which
    // spares the lookup of a preorder position's node.
    // (lane k also loads node_off[min(k, n_req)], so that a node's request offset is a
    // lane exchange rather than a dependent load)
    const int li = (int)threadIdx.x & (kNodesPerBlock - 1);
    const int pos = n0 + (li < nn ? li : 0);
    const int i_req = p.blob[p.o_req + pos];
    int mine = pos;
    if (p.pre) {
        const int nof = p.blob[p.o_node_off + min((int)threadIdx.x & 63, p.n_req)];
        const int nsh = __shfl(nof, i_req & 63);
        mine = (i_req < 64 ? nsh : p.blob[p.o_node_off + i_req]) + p.blob[p.o_dfs + pos];
    }
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

// Depth-first variant (bf16, paths of at most 16 nodes). One block walks one request's
// tree in preorder for one layer and 2048 channels; each thread keeps, for its 8
// channels, the x entries of the current root path (after the three history entries)
// in registers, so every x row is read from memory exactly once. A node at depth d has
// the window (ext[d], ext[d+1], ext[d+2], x_node) with ext = (history, path by depth);
// taps, accumulation order, activation and cast are those of conv_kernel. With PH the
// block first publishes the pending path into its slice of the history (which no other
// block reads) and takes the three entries from registers; requests without nodes in
// this iteration only publish.
constexpr int kDfsWin = 512;  // preorder positions staged in LDS at a time
constexpr int kDfsGroup = 4;  // nodes whose rows are loaded one group ahead

struct ConvDfsParams {
    const int32_t* blob;
    int32_t o_node_off, o_pre_row, o_pre_depth;
    int32_t n_req, total_rows, n_layers, channels, n_cchunks, act;
    const uint16_t* x;
    const uint16_t* hist;
    const float* w;
    const float* bias;
    uint16_t* y;
};

__device__ __forceinline__ void dfs_pin(uint4& a) {
    asm volatile("" : "+v"(a.x), "+v"(a.y), "+v"(a.z), "+v"(a.w));
}

// The window's three older entries for a node at depth d (< DD), and the node's own
// entry recorded at depth d: a chain of uniform branches to static register indices.
// The empty asm statements keep the compiler from merging the branches into one
// indexed access, which would move the array to scratch memory.
template <int DD, int D = 0>
__device__ __forceinline__ void dfs_taps(int d, uint4 (&ext)[DD + 3], const uint4 xt, uint4& t0, uint4& t1,
                                         uint4& t2) {
    if constexpr (D + 1 < DD) {
        if (d != D) {
            dfs_taps<DD, D + 1>(d, ext, xt, t0, t1, t2);
            return;
        }
    }
    t0 = ext[D];
    t1 = ext[D + 1];
    t2 = ext[D + 2];
    ext[3 + D] = xt;
    dfs_pin(t0);
    dfs_pin(t1);
    dfs_pin(t2);
    asm volatile("" ::"n"(D) : "memory");
}

template <int DD, bool PH>
__global__ __launch_bounds__(256) void conv_dfs_kernel(ConvDfsParams p, HistPend hp) {
    int t = xcd_remap(blockIdx.x, gridDim.x);
    const int cc = t % p.n_cchunks;
    t /= p.n_cchunks;
    const int r = t % p.n_req;
    const int l = t / p.n_req;
    const int base = p.blob[p.o_node_off + r];
    const int N = p.blob[p.o_node_off + r + 1] - base;
    const int tid = (int)threadIdx.x;
    const int c0ch = (cc * 256 + tid) * 8;
    const bool has_c = c0ch < p.channels;
    const int c = has_c ? c0ch : p.channels - 8;
    uint4 ext[DD + 3];
    const uint16_t* hr = p.hist + ((long)r * p.n_layers + l) * 3 * p.channels + c;
    const int plen = PH ? pend_hist_len(hp, r) : 0;  // uniform
    if (plen > 0) {
        const uint16_t* hrl = p.hist + ((long)r * p.n_layers + l) * 3 * p.channels;
#pragma unroll
        for (int e = 0; e < 3; ++e)
            ext[e] = *reinterpret_cast<const uint4*>(pend_hist_src<uint16_t>(hp, hrl, r, l, plen, e, p.channels, c));
        if (has_c) {
            uint16_t* hw = static_cast<uint16_t*>(hp.hist) + ((long)r * p.n_layers + l) * 3 * p.channels + c;
#pragma unroll
            for (int e = 0; e < 3; ++e) *reinterpret_cast<uint4*>(hw + (long)e * p.channels) = ext[e];
        }
    } else if (N > 0) {
#pragma unroll
        for (int e = 0; e < 3; ++e) ext[e] = *reinterpret_cast<const uint4*>(hr + (long)e * p.channels);
    }
    if (N <= 0) return;  // uniform over the block
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
#pragma unroll
    for (int e = 3; e < DD + 3; ++e) ext[e] = make_uint4(0, 0, 0, 0);  // written before read in preorder
    const uint16_t* xl = p.x + (long)l * p.total_rows * p.channels + c;
    uint16_t* yl = p.y + (long)l * p.total_rows * p.channels + c;
    const int32_t* prow = p.blob + p.o_pre_row + base;
    const int32_t* pdep = p.blob + p.o_pre_depth + base;
    __shared__ int2 info[kDfsWin];  // (row, depth) of preorder positions w0 ..
    for (int w0 = 0; w0 < N; w0 += kDfsWin) {
        const int nw = min(kDfsWin, N - w0);
        __syncthreads();  // the previous window's entries have been read
        for (int i = tid; i < nw; i += 256) info[i] = make_int2(prow[w0 + i], pdep[w0 + i]);
        __syncthreads();
        uint4 buf[2][kDfsGroup];
        auto issue = [&](int g, uint4 (&b)[kDfsGroup]) __attribute__((always_inline)) {
#pragma unroll
            for (int i = 0; i < kDfsGroup; ++i) {
                const int row = __builtin_amdgcn_readfirstlane(info[min(g * kDfsGroup + i, nw - 1)].x);
                b[i] = *reinterpret_cast<const uint4*>(xl + (long)row * p.channels);
            }
        };
        auto compute = [&](int g, const uint4 (&b)[kDfsGroup]) __attribute__((always_inline)) {
#pragma unroll
            for (int i = 0; i < kDfsGroup; ++i) {
                const int j = g * kDfsGroup + i;
                if (j >= nw) break;  // uniform
                const int2 in = info[j];
                const int row = __builtin_amdgcn_readfirstlane(in.x);
                const int d = __builtin_amdgcn_readfirstlane(in.y);
                uint4 tp[4];
                dfs_taps<DD>(d, ext, b[i], tp[0], tp[1], tp[2]);
                tp[3] = b[i];
                float acc[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) acc[e] = b0[e];
#pragma unroll
                for (int tap = 0; tap < 4; ++tap) {
                    float xv[8];
                    Vec8<1>::unpack(tp[tap], xv);
#pragma unroll
                    for (int e = 0; e < 8; ++e) acc[e] = __builtin_fmaf(wt[4 * e + tap], xv[e], acc[e]);
                }
                if (p.act == 1) {
#pragma unroll
                    for (int e = 0; e < 8; ++e) acc[e] = acc[e] * __builtin_amdgcn_rcpf(1.f + __expf(-acc[e]));
                }
                if (has_c) Vec8<1>::st(yl + (long)row * p.channels, acc);
            }
        };
        const int ng = (nw + kDfsGroup - 1) / kDfsGroup;
        issue(0, buf[0]);
        for (int g = 0; g < ng; g += 2) {
            if (g + 1 < ng) issue(g + 1, buf[1]);
            compute(g, buf[0]);
            if (g + 1 < ng) {
                if (g + 2 < ng) issue(g + 2, buf[0]);
                compute(g + 1, buf[1]);
            }
        }
    }
}

}  // namespace

hipError_t launch_conv(const lumo_gdn_dims& d, const lumo_tree_desc& desc, const ConvArgs& a, hipStream_t s,
                       const ConvPendArgs* pend) {
    const lumo_plan& pl = desc.plan;
    const int n_cchunks = (a.channels + 2047) / 2048;
    HistPend hq{};
    if (pend) {
        const lumo_plan& pp = pend->desc->plan;
        hq.blob = pend->desc->blob;
        hq.o_node_off = pp.o_node_off;
        hq.o_row = pp.o_row;
        hq.total_rows = pp.total_rows;
        hq.max_path = pend->max_path;
        hq.path_out = pend->path_out;
        hq.path_len = pend->path_len;
        hq.x_prev = pend->x_prev;
        hq.hist = const_cast<void*>(a.hist);
    }
    // The depth-first walk reads every x row once but runs one block per (request, layer,
    // channel block), each walking its request's nodes in sequence: it is chosen when
    // that gives at least four blocks per CU; otherwise the run kernel's parallelism over
    // node runs wins (measured: one request or one layer of 128-256-node trees).
    const long dfs_blocks = (long)d.n_req * d.n_layers * n_cchunks;
    const bool dfs = d.op_dtype == LUMO_BF16 && pl.max_depth <= 16 && dfs_blocks >= 4 * 256;
    if (pend && !dfs) {  // publish first, then the run kernel reads the history
        const long hb = (long)d.n_req * d.n_layers * n_cchunks;
        if (d.op_dtype == LUMO_BF16)
            hipLaunchKernelGGL(hist_pend_kernel<1>, dim3((unsigned)hb), dim3(256), 0, s, hq, d.n_layers, a.channels,
                               n_cchunks);
        else
            hipLaunchKernelGGL(hist_pend_kernel<0>, dim3((unsigned)hb), dim3(256), 0, s, hq, d.n_layers, a.channels,
                               n_cchunks);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (dfs && (pl.total_nodes > 0 || pend)) {  // with pend, requests without nodes still publish
        ConvDfsParams q;
        q.blob = desc.blob;
        q.o_node_off = pl.o_node_off;
        q.o_pre_row = pl.o_pre_row;
        q.o_pre_depth = pl.o_pre_depth;
        q.n_req = d.n_req;
        q.total_rows = pl.total_rows;
        q.n_layers = d.n_layers;
        q.channels = a.channels;
        q.n_cchunks = n_cchunks;
        q.act = a.act;
        q.x = static_cast<const uint16_t*>(a.x);
        q.hist = static_cast<const uint16_t*>(a.hist);
        q.w = a.w;
        q.bias = a.bias;
        q.y = static_cast<uint16_t*>(a.y);
        const dim3 grid((unsigned)dfs_blocks);
        if (pl.max_depth <= 8) {
            if (pend)
                hipLaunchKernelGGL((conv_dfs_kernel<8, true>), grid, dim3(256), 0, s, q, hq);
            else
                hipLaunchKernelGGL((conv_dfs_kernel<8, false>), grid, dim3(256), 0, s, q, hq);
        } else {
            if (pend)
                hipLaunchKernelGGL((conv_dfs_kernel<16, true>), grid, dim3(256), 0, s, q, hq);
            else
                hipLaunchKernelGGL((conv_dfs_kernel<16, false>), grid, dim3(256), 0, s, q, hq);
        }
        return hipGetLastError();
    }
    if (pl.total_nodes == 0) return hipSuccess;
    ConvParams p;
    p.blob = desc.blob;
    p.o_req = pl.o_req;
    p.o_row = pl.o_row;
    p.o_conv_src = pl.o_conv_src;
    p.o_node_off = pl.o_node_off;
    p.o_dfs = pl.o_dfs;
    p.n_req = d.n_req;
    p.total_nodes = pl.total_nodes;
    p.total_rows = pl.total_rows;
    p.n_layers = d.n_layers;
    p.channels = a.channels;
    p.n_cchunks = n_cchunks;
    p.act = a.act;
    p.x = a.x;
    p.hist = a.hist;
    p.w = a.w;
    p.bias = a.bias;
    p.y = a.y;
    // runs of 32 nodes, halved (down to 4) while the grid has fewer than four blocks per
    // CU: a block's node batches are loaded one after the other, so small grids (one
    // layer of a batch) finish sooner with more, shorter runs
    int run = kNodesPerBlock;
    while (run > 4 && (long)d.n_layers * n_cchunks * ((pl.total_nodes + run - 1) / run) < 4 * 256) run /= 2;
    p.run = run;
    p.pre = run == kNodesPerBlock;
    const long blocks = (long)d.n_layers * n_cchunks * ((pl.total_nodes + run - 1) / run);
    if (d.op_dtype == LUMO_BF16)
        hipLaunchKernelGGL(conv_kernel<1>, dim3((unsigned)blocks), dim3(256), 0, s, p);
    else
        hipLaunchKernelGGL(conv_kernel<0>, dim3((unsigned)blocks), dim3(256), 0, s, p);
    return hipGetLastError();
}

}  // namespace lumo
