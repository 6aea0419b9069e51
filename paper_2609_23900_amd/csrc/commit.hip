// Accepted-path publication (LumoTree Alg. 1 publication, Alg. 2 replay, Sec. V-A).
//
// Fixed-shape launches, all driven by device data only (no host path list):
//   1. path + history kernel  accepted node -> root-first path and its length
//                     (bit-exact); conv history <- last three of (history, x rows of
//                     the path). Without conv operands, the path kernel alone.
//   2. replay kernel  one wavefront per (request, layer, value head, value tile):
//                     load the pre-tree state tile, apply the recorded updates of the
//                     path with the same row update the verifier uses, store in place;
//                     before the loop the path's first key rows are copied to LDS
//                     (direct global-to-LDS loads, in flight with the state load) and
//                     its rows, decays, betas and value entries are fetched into lanes.
//                     Skipped when the state is NULL (publication deferred).
// Empty or invalid paths leave the state and the history untouched.
#include "device_common.h"
#include "internal.h"
#include "commit.h"

namespace lumo {
namespace {

struct PathParams {
    const int32_t* blob;
    int32_t o_node_off, o_parent, o_depth;
    int32_t n_req, max_path;
    const int32_t* accepted;
    int32_t* path_out;
    int32_t* path_len;
};

__global__ __launch_bounds__(256) void path_kernel(PathParams p) {
    const int r = blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= p.n_req) return;
    const int base = p.blob[p.o_node_off + r];
    const int n = p.blob[p.o_node_off + r + 1] - base;
    const int a = p.accepted[r];
    int len;
    if (a < -1 || a >= n) {
        len = -1;
    } else if (a == -1) {
        len = 0;
    } else {
        len = p.blob[p.o_depth + base + a] + 1;
        if (len > p.max_path) len = -1;
    }
    int32_t* po = p.path_out + (long)r * p.max_path;
    for (int i = 0; i < p.max_path; ++i) po[i] = -1;
    int x = a;
    for (int i = len - 1; i >= 0; --i) {  // len <= depth + 1, so the walk ends at the root
        po[i] = x;
        x = p.blob[p.o_parent + base + x];
    }
    p.path_len[r] = len;
}

struct ReplayParams {
    const int32_t* blob;
    int32_t o_node_off, o_row;
    int32_t max_path, n_layers, total_rows, h_k, h_v, d_v, group, n_vtiles;
    PrepArgs prep;  // operand preparation of the path's k, g, beta
};

// Path entries whose key row, row, decay, beta and value are fetched before the loop.
constexpr int kPrefetch = 16;

template <int DK, int OPT> struct KeyRows {
    using T = typename Op<OPT>::T;
    static constexpr int kSeg = DK * (int)sizeof(T) / 16;                  // 16-byte segments per row
    static constexpr int kSlots = (kPrefetch * kSeg + 63) / 64 * 64;      // whole wave copies
};

// One 16-byte segment of a key row as floats (4 fp32 or 8 bf16 values).
template <int OPT> __device__ __forceinline__ void unpack_seg(const uint4 w, float (&f)[16 / (OPT ? 2 : 4)]);
template <> __device__ __forceinline__ void unpack_seg<0>(const uint4 w, float (&f)[4]) {
    f[0] = __uint_as_float(w.x); f[1] = __uint_as_float(w.y); f[2] = __uint_as_float(w.z); f[3] = __uint_as_float(w.w);
}
template <> __device__ __forceinline__ void unpack_seg<1>(const uint4 w, float (&f)[8]) {
    f[0] = bf16_lo(w.x); f[1] = bf16_hi(w.x); f[2] = bf16_lo(w.y); f[3] = bf16_hi(w.y);
    f[4] = bf16_lo(w.z); f[5] = bf16_hi(w.z); f[6] = bf16_lo(w.w); f[7] = bf16_hi(w.w);
}

// The verifier's row update (gdn_row_update: same operations in the same order, so
// the result is bitwise identical) with the key row read from LDS, 32 elements at a
// time (the compiler barrier keeps it from hoisting the whole row into registers).
// ks scales the key (1/|k| with query/key normalisation, else exactly 1).
template <int DK, int OPT>
__device__ __forceinline__ void row_update_lds(float (&S)[DK], const uint4* kr, float vj, float alpha, float beta,
                                               float ks) {
    constexpr int E = 16 / (int)sizeof(typename Op<OPT>::T);  // elements per 16-byte segment
    constexpr int C = DK < 32 ? DK : 32;
    Dot4 u;
#pragma unroll
    for (int c0 = 0; c0 < DK; c0 += C) {
        asm volatile("" ::: "memory");
#pragma unroll
        for (int c = c0; c < c0 + C; c += E) {
            float kf[E];
            unpack_seg<OPT>(kr[c / E], kf);
#pragma unroll
            for (int i = 0; i < E; ++i) u.add(c + i, S[c + i], kf[i]);
        }
    }
    const float delta = beta * __builtin_fmaf(-alpha, u.sum() * ks, vj) * ks;
#pragma unroll
    for (int c0 = 0; c0 < DK; c0 += C) {
        asm volatile("" ::: "memory");
#pragma unroll
        for (int c = c0; c < c0 + C; c += E) {
            float kf[E];
            unpack_seg<OPT>(kr[c / E], kf);
#pragma unroll
            for (int i = 0; i < E; ++i) S[c + i] = __builtin_fmaf(delta, kf[i], alpha * S[c + i]);
        }
    }
}

// Entries e0 .. e0 + kPrefetch - 1 of the path: lane e receives entry e0 + e's decay
// and beta; its key row and the tile's 64 values go to LDS (direct global-to-LDS
// copies). Lanes and slots past the path repeat its last entry.
template <int DK, int OPT>
__device__ __forceinline__ void replay_stage(const ReplayParams& p, const typename Op<OPT>::T* __restrict__ k,
                                             const typename Op<OPT>::T* __restrict__ v, const float* __restrict__ g,
                                             const float* __restrict__ beta, const int32_t* path, int base, int len,
                                             int e0, int l, int h, int hk, int vt, int lane, uint4* krows,
                                             uint4* vrows, float& apre, float& bpre) {
    using T = typename Op<OPT>::T;
    using KR = KeyRows<DK, OPT>;
    constexpr int E = 16 / (int)sizeof(T);
    constexpr int kVSeg = 64 / E;
    const int ne = min(len - e0, kPrefetch);
    const int prow = p.blob[p.o_row + base + path[e0 + min(lane, ne - 1)]];
    const long gl = ((long)l * p.total_rows + prow) * p.h_v + h;
    float gv = g[gl], bv = beta[gl];
    if (p.prep.flags & LUMO_PREP_RAW_GATES) {
        const int lh = l * p.h_v + h;
        gv = raw_log_alpha(gv, p.prep.a_log[lh], p.prep.dt_bias[lh]);
        bv = raw_beta(bv);
    }
    apre = __expf(gv);
    bpre = bv;
#pragma unroll
    for (int i = 0; i < KR::kSlots / 64; ++i) {
        const int sl = 64 * i + lane;
        const int re = __shfl(prow, min(sl / KR::kSeg, ne - 1));
        const T* kr = k + (((long)l * p.total_rows + re) * p.h_k + hk) * DK;
        __builtin_amdgcn_global_load_lds(reinterpret_cast<const uint4*>(kr) + sl % KR::kSeg,
                                         (__attribute__((address_space(3))) void*)&krows[64 * i], 16, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < kPrefetch * kVSeg / 64; ++i) {
        const int sl = 64 * i + lane;
        const int re = __shfl(prow, min(sl / kVSeg, ne - 1));
        const int c = min(vt * 64 + (sl % kVSeg) * E, p.d_v - E);  // columns past d_v: any valid segment
        const T* vr = v + (((long)l * p.total_rows + re) * p.h_v + h) * p.d_v + c;
        __builtin_amdgcn_global_load_lds(reinterpret_cast<const uint4*>(vr),
                                         (__attribute__((address_space(3))) void*)&vrows[64 * i], 16, 0, 0);
    }
}

template <int DK, int OPT>
__global__ __launch_bounds__(64, 2) void replay_kernel(ReplayParams p, const typename Op<OPT>::T* __restrict__ k,
                                                   const typename Op<OPT>::T* __restrict__ v,
                                                   const float* __restrict__ g, const float* __restrict__ beta,
                                                   float* __restrict__ state, const int32_t* __restrict__ path_out,
                                                   const int32_t* __restrict__ path_len) {
    int t = xcd_remap(blockIdx.x, gridDim.x);
    const int vt = t % p.n_vtiles;
    t /= p.n_vtiles;
    const int h = t % p.h_v;
    t /= p.h_v;
    const int l = t % p.n_layers;
    const int r = t / p.n_layers;
    using T = typename Op<OPT>::T;
    using KR = KeyRows<DK, OPT>;
    constexpr int E = 16 / (int)sizeof(T);          // elements per 16-byte segment
    constexpr int kVSeg = 64 / E;                   // segments of one entry's 64 values
    constexpr int kVSlots = kPrefetch * kVSeg;      // 128 or 256: whole wave copies
    __shared__ uint4 krows[KR::kSlots];
    __shared__ uint4 vrows[kVSlots];
    const int len = path_len[r];
    if (len <= 0) return;
    const int lane = (int)threadIdx.x;
    const int j = vt * 64 + lane;
    const bool act = j < p.d_v;
    const int jc = act ? j : p.d_v - 1;
    const int hk = h / p.group;
    const int base = p.blob[p.o_node_off + r];
    const long mat = (long)DK * p.d_v;
    float* st = state + (((long)r * p.n_layers + l) * p.h_v + h) * mat;
    const int32_t* path = path_out + (long)r * p.max_path;
    float apre, bpre;
    replay_stage<DK, OPT>(p, k, v, g, beta, path, base, len, 0, l, h, hk, vt, lane, krows, vrows, apre, bpre);
    float S[DK];
#pragma unroll
    for (int i = 0; i < DK; ++i) S[i] = (st + (long)i * p.d_v)[jc];  // uniform row base + lane offset
    const T* vl = reinterpret_cast<const T*>(vrows);
    for (int e0 = 0; e0 < len; e0 += kPrefetch) {
        if (e0 > 0)  // paths longer than kPrefetch: the previous block has been consumed
            replay_stage<DK, OPT>(p, k, v, g, beta, path, base, len, e0, l, h, hk, vt, lane, krows, vrows, apre, bpre);
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // the staged rows have landed in LDS
        const int ne = min(len - e0, kPrefetch);
        float kspre = 1.f;  // lane e: 1/sqrt(|k|^2 + eps) of entry e's key (normalisation)
        if (p.prep.flags & LUMO_PREP_QK_NORM) {
            constexpr int E = 16 / (int)sizeof(T);
            const uint4* kr = krows + min(lane, ne - 1) * KR::kSeg;
            float ss = 0.f;
            for (int sg = 0; sg < KR::kSeg; ++sg) {
                float f[E];
                unpack_seg<OPT>(kr[sg], f);
#pragma unroll
                for (int i = 0; i < E; ++i) ss = __builtin_fmaf(f[i], f[i], ss);
            }
            kspre = __builtin_amdgcn_rsqf(ss + p.prep.qk_eps);
        }
        for (int e = 0; e < ne; ++e) {
            const float ae = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(apre), e));
            const float be = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(bpre), e));
            const float ke = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(kspre), e));
            row_update_lds<DK, OPT>(S, krows + e * KR::kSeg, Op<OPT>::ld(vl, e * 64 + lane), ae, be, ke);
        }
    }
    if (act) {
#pragma unroll
        for (int i = 0; i < DK; ++i) (st + (long)i * p.d_v)[j] = S[i];
    }
}

struct HistParams {
    const int32_t* blob;
    int32_t o_node_off, o_row;
    int32_t n_layers, total_rows, channels, n_cchunks;
    const void* x;
    void* hist;
};

// Path derivation and conv-history publication in one launch (with conv operands).
// Every block of request r derives r's path length with the path kernel's rule; the
// block (r, layer 0, channel chunk 0) also writes path_out and path_len. The history
// needs only the path's last three nodes: the accepted node and its two nearest
// ancestors, read straight from the parent table. hist_rl is the history of (r, l)
// ([3][channels]), x_l the rows of layer l ([rows][channels]).
template <class T>
__device__ __forceinline__ void path_hist_block(const PathParams& pp, const HistParams& p, int r, int l, int cc,
                                                T* hist_rl, const T* x_l) {
    const int base = p.blob[p.o_node_off + r];
    const int n = p.blob[p.o_node_off + r + 1] - base;
    const int a = pp.accepted[r];
    int len;
    if (a < -1 || a >= n) {
        len = -1;
    } else if (a == -1) {
        len = 0;
    } else {
        len = pp.blob[pp.o_depth + base + a] + 1;
        if (len > pp.max_path) len = -1;
    }
    if (l == 0 && cc == 0 && threadIdx.x < 64) {
        int32_t* po = pp.path_out + (long)r * pp.max_path;
        for (int i = (int)threadIdx.x; i < pp.max_path; i += 64)
            if (i >= len) po[i] = -1;
        if (threadIdx.x == 0) {
            int x = a;
            for (int i = len - 1; i >= 0; --i) {  // len <= depth + 1: the walk ends at the root
                po[i] = x;
                x = pp.blob[pp.o_parent + base + x];
            }
            pp.path_len[r] = len;
        }
    }
    if (len <= 0) return;
    const int c = (cc * 256 + (int)threadIdx.x) * 8;
    if (c >= p.channels) return;
    // entry e of the new history is entry len + e of (history, x rows of the path); for
    // len + e >= 3 that is path node len + e - 3, the (2 - e)-th ancestor of the accepted node
    int node[3];
    node[2] = a;
    node[1] = len >= 2 ? pp.blob[pp.o_parent + base + a] : -1;
    node[0] = len >= 3 ? pp.blob[pp.o_parent + base + node[1]] : -1;
    const T* src[3];
#pragma unroll
    for (int e = 0; e < 3; ++e) {
        const int pos = len + e;
        src[e] = pos < 3 ? hist_rl + (long)pos * p.channels + c
                         : x_l + (long)p.blob[p.o_row + base + node[e]] * p.channels + c;
    }
    constexpr int W = 16 / sizeof(T) >= 8 ? 1 : 2;  // 16-byte pieces per 8 channels
#pragma unroll
    for (int w = 0; w < W; ++w) {  // each piece read whole before it is overwritten
        const uint4 v0 = reinterpret_cast<const uint4*>(src[0])[w];
        const uint4 v1 = reinterpret_cast<const uint4*>(src[1])[w];
        const uint4 v2 = reinterpret_cast<const uint4*>(src[2])[w];
        reinterpret_cast<uint4*>(hist_rl + c)[w] = v0;
        reinterpret_cast<uint4*>(hist_rl + (long)p.channels + c)[w] = v1;
        reinterpret_cast<uint4*>(hist_rl + 2L * p.channels + c)[w] = v2;
    }
}

// Stacked operands: history [n_req][n_layers][3][channels], x [n_layers][rows][channels].
template <int OPT>
__global__ __launch_bounds__(256) void path_hist_kernel(PathParams pp, HistParams p) {
    using T = typename Op<OPT>::T;
    const int cc = blockIdx.x % p.n_cchunks;
    const int l = (blockIdx.x / p.n_cchunks) % p.n_layers;
    const int r = blockIdx.x / (p.n_cchunks * p.n_layers);
    T* hist = static_cast<T*>(p.hist) + (((long)r * p.n_layers + l) * 3) * p.channels;
    const T* x = static_cast<const T*>(p.x) + (long)l * p.total_rows * p.channels;
    path_hist_block<T>(pp, p, r, l, cc, hist, x);
}

// Each layer's own buffers, passed by value: history [n_req][3][channels] and
// x [rows][channels] of layer l.
struct LayerTable {
    const void* x[kMaxLayerTable];
    void* hist[kMaxLayerTable];
};

template <int OPT>
__global__ __launch_bounds__(256) void path_hist_layers_kernel(PathParams pp, HistParams p, LayerTable lt) {
    using T = typename Op<OPT>::T;
    const int cc = blockIdx.x % p.n_cchunks;
    const int l = (blockIdx.x / p.n_cchunks) % p.n_layers;
    const int r = blockIdx.x / (p.n_cchunks * p.n_layers);
    T* hist = static_cast<T*>(lt.hist[l]) + (long)r * 3 * p.channels;
    path_hist_block<T>(pp, p, r, l, cc, hist, static_cast<const T*>(lt.x[l]));
}

template <int DK, int OPT>
void launch_replay_dk(dim3 grid, hipStream_t s, const ReplayParams& p, const CommitArgs& a) {
    using T = typename Op<OPT>::T;
    hipLaunchKernelGGL((replay_kernel<DK, OPT>), grid, dim3(64), 0, s, p, static_cast<const T*>(a.k),
                       static_cast<const T*>(a.v), a.g, a.beta, a.state, a.path_out, a.path_len);
}

template <int OPT>
hipError_t launch_replay(int dk, dim3 grid, hipStream_t s, const ReplayParams& p, const CommitArgs& a) {
    switch (dk) {
        case 16: launch_replay_dk<16, OPT>(grid, s, p, a); break;
        case 32: launch_replay_dk<32, OPT>(grid, s, p, a); break;
        case 64: launch_replay_dk<64, OPT>(grid, s, p, a); break;
        default: launch_replay_dk<128, OPT>(grid, s, p, a); break;
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_commit(const lumo_gdn_dims& d, const lumo_tree_desc& desc, const CommitArgs& a, hipStream_t s) {
    const lumo_plan& pl = desc.plan;
    if (d.n_req == 0) return hipSuccess;
    PathParams pp{desc.blob, pl.o_node_off, pl.o_parent, pl.o_depth, d.n_req, a.max_path,
                  a.accepted, a.path_out, a.path_len};
    const bool conv = a.x && a.conv_hist;
    if (conv) {  // path and history together (the replay only needs the path, written first)
        HistParams hp;
        hp.blob = desc.blob;
        hp.o_node_off = pl.o_node_off;
        hp.o_row = pl.o_row;
        hp.n_layers = d.n_layers;
        hp.total_rows = pl.total_rows;
        hp.channels = a.channels;
        hp.n_cchunks = (a.channels + 2047) / 2048;
        hp.x = a.x;
        hp.hist = a.conv_hist;
        const long hb = (long)d.n_req * d.n_layers * hp.n_cchunks;
        if (d.op_dtype == LUMO_BF16)
            hipLaunchKernelGGL(path_hist_kernel<1>, dim3((unsigned)hb), dim3(256), 0, s, pp, hp);
        else
            hipLaunchKernelGGL(path_hist_kernel<0>, dim3((unsigned)hb), dim3(256), 0, s, pp, hp);
    } else {
        hipLaunchKernelGGL(path_kernel, dim3((d.n_req + 255) / 256), dim3(256), 0, s, pp);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;

    if (a.state) {  // NULL: the replay is deferred to the next verification
    ReplayParams rp;
    rp.blob = desc.blob;
    rp.o_node_off = pl.o_node_off;
    rp.o_row = pl.o_row;
    rp.max_path = a.max_path;
    rp.n_layers = d.n_layers;
    rp.total_rows = pl.total_rows;
    rp.h_k = d.h_k;
    rp.h_v = d.h_v;
    rp.d_v = d.d_v;
    rp.group = d.h_v / d.h_k;
    rp.n_vtiles = (d.d_v + 63) / 64;
    rp.prep = a.prep;
    const long blocks = (long)d.n_req * d.n_layers * d.h_v * rp.n_vtiles;
    e = d.op_dtype == LUMO_BF16 ? launch_replay<1>(d.d_k, dim3((unsigned)blocks), s, rp, a)
                                : launch_replay<0>(d.d_k, dim3((unsigned)blocks), s, rp, a);
    if (e != hipSuccess) return e;
    }

    return e;
}

hipError_t launch_commit_hist_layers(const lumo_gdn_dims& d, const lumo_tree_desc& desc, const CommitArgs& a,
                                     const void* const* x_layers, void* const* hist_layers, hipStream_t s) {
    const lumo_plan& pl = desc.plan;
    if (d.n_req == 0) return hipSuccess;
    if (d.n_layers > kMaxLayerTable) return hipErrorInvalidValue;
    PathParams pp{desc.blob, pl.o_node_off, pl.o_parent, pl.o_depth, d.n_req, a.max_path,
                  a.accepted, a.path_out, a.path_len};
    HistParams hp;
    hp.blob = desc.blob;
    hp.o_node_off = pl.o_node_off;
    hp.o_row = pl.o_row;
    hp.n_layers = d.n_layers;
    hp.total_rows = pl.total_rows;
    hp.channels = a.channels;
    hp.n_cchunks = (a.channels + 2047) / 2048;
    hp.x = nullptr;
    hp.hist = nullptr;
    LayerTable lt{};
    for (int l = 0; l < d.n_layers; ++l) {
        lt.x[l] = x_layers[l];
        lt.hist[l] = hist_layers[l];
    }
    const long hb = (long)d.n_req * d.n_layers * hp.n_cchunks;
    if (d.op_dtype == LUMO_BF16)
        hipLaunchKernelGGL(path_hist_layers_kernel<1>, dim3((unsigned)hb), dim3(256), 0, s, pp, hp, lt);
    else
        hipLaunchKernelGGL(path_hist_layers_kernel<0>, dim3((unsigned)hb), dim3(256), 0, s, pp, hp, lt);
    return hipGetLastError();
}

}  // namespace lumo
