// Accepted-path publication (LumoTree Alg. 1 publication, Alg. 2 replay, Sec. V-A).
//
// Three fixed-shape launches, all driven by device data only (no host path list):
//   1. path kernel    accepted node -> root-first path and its length (bit-exact)
//   2. replay kernel  one wavefront per (request, layer, value head, value tile):
//                     load the pre-tree state tile, apply the recorded updates of the
//                     path with the same row update the verifier uses, store in place;
//                     the path's rows and value entries are fetched before the loop,
//                     the wave-uniform key rows are read with scalar loads
//   3. history kernel conv history <- last three of (history, x rows of the path)
// Empty or invalid paths leave the state and the history untouched.
#include "device_common.h"
#include "internal.h"
#include "launch.h"

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
};

// Path entries whose row and value are prefetched before the update loop.
constexpr int kPrefetch = 16;

// One replayed update (the verifier's row update) for path entry e.
template <int DK, int OPT>
__device__ __forceinline__ void replay_step(float (&S)[DK], const typename Op<OPT>::T* __restrict__ k,
                                            const float* __restrict__ g, const float* __restrict__ beta,
                                            const ReplayParams& p, int l, int h, int hk, int row, float vj) {
    const long gi = ((long)l * p.total_rows + row) * p.h_v + h;
    const long ki = (((long)l * p.total_rows + row) * p.h_k + hk) * DK;
    gdn_row_update<DK, OPT>(S, k + ki, vj, __expf(g[gi]), beta[gi]);
}

template <int DK, int OPT>
__global__ __launch_bounds__(64) void replay_kernel(ReplayParams p, const typename Op<OPT>::T* __restrict__ k,
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
    // row of path entry `lane` (lanes past the path read the root's row)
    const int prow = p.blob[p.o_row + base + path[lane < len ? lane : 0]];
    float vpre[kPrefetch];
#pragma unroll
    for (int e = 0; e < kPrefetch; ++e) {
        const int re = __builtin_amdgcn_readlane(prow, e);  // wave-uniform row
        vpre[e] = Op<OPT>::ld(v, (((long)l * p.total_rows + re) * p.h_v + h) * p.d_v + jc);
    }
    float S[DK];
#pragma unroll
    for (int i = 0; i < DK; ++i) S[i] = st[(long)i * p.d_v + jc];
    for (int e = 0; e < len; ++e) {
        const int re = e < 64 ? __builtin_amdgcn_readlane(prow, e) : p.blob[p.o_row + base + path[e]];
        const float vj = e < kPrefetch ? vpre[0]
                                       : Op<OPT>::ld(v, (((long)l * p.total_rows + re) * p.h_v + h) * p.d_v + jc);
        replay_step<DK, OPT>(S, k, g, beta, p, l, h, hk, re, vj);
#pragma unroll
        for (int i = 0; i + 1 < kPrefetch; ++i) vpre[i] = vpre[i + 1];  // next entry's value to slot 0
    }
    if (act) {
#pragma unroll
        for (int i = 0; i < DK; ++i) st[(long)i * p.d_v + j] = S[i];
    }
}

struct HistParams {
    const int32_t* blob;
    int32_t o_node_off, o_row;
    const int32_t* path_out;
    const int32_t* path_len;
    int32_t max_path, n_layers, total_rows, channels, n_cchunks;
    const void* x;
    void* hist;
};

// 8 channels per thread: 16 bytes of bf16, 32 bytes of fp32.
template <int OPT>
__global__ __launch_bounds__(256) void hist_kernel(HistParams p) {
    using T = typename Op<OPT>::T;
    const int cc = blockIdx.x % p.n_cchunks;
    const int l = (blockIdx.x / p.n_cchunks) % p.n_layers;
    const int r = blockIdx.x / (p.n_cchunks * p.n_layers);
    const int len = p.path_len[r];
    if (len <= 0) return;
    const int c = (cc * 256 + (int)threadIdx.x) * 8;
    if (c >= p.channels) return;
    const int base = p.blob[p.o_node_off + r];
    T* hist = static_cast<T*>(p.hist) + (((long)r * p.n_layers + l) * 3) * p.channels;
    const T* x = static_cast<const T*>(p.x);
    constexpr int W = 16 / sizeof(T) >= 8 ? 1 : 2;  // uint4 loads per 8 channels
    uint4 val[3][W];
#pragma unroll
    for (int e = 0; e < 3; ++e) {
        const int pos = len + e;  // entry e of the last three of (3 + len) entries
        const T* src;
        if (pos < 3) {
            src = hist + (long)pos * p.channels + c;
        } else {
            const int row = p.blob[p.o_row + base + p.path_out[(long)r * p.max_path + pos - 3]];
            src = x + ((long)l * p.total_rows + row) * p.channels + c;
        }
#pragma unroll
        for (int w = 0; w < W; ++w) val[e][w] = reinterpret_cast<const uint4*>(src)[w];
    }
#pragma unroll
    for (int e = 0; e < 3; ++e)
#pragma unroll
        for (int w = 0; w < W; ++w) reinterpret_cast<uint4*>(hist + (long)e * p.channels + c)[w] = val[e][w];
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
    hipLaunchKernelGGL(path_kernel, dim3((d.n_req + 255) / 256), dim3(256), 0, s, pp);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;

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
    const long blocks = (long)d.n_req * d.n_layers * d.h_v * rp.n_vtiles;
    e = d.op_dtype == LUMO_BF16 ? launch_replay<1>(d.d_k, dim3((unsigned)blocks), s, rp, a)
                                : launch_replay<0>(d.d_k, dim3((unsigned)blocks), s, rp, a);
    if (e != hipSuccess) return e;

    if (a.x && a.conv_hist) {
        HistParams hp;
        hp.blob = desc.blob;
        hp.o_node_off = pl.o_node_off;
        hp.o_row = pl.o_row;
        hp.path_out = a.path_out;
        hp.path_len = a.path_len;
        hp.max_path = a.max_path;
        hp.n_layers = d.n_layers;
        hp.total_rows = pl.total_rows;
        hp.channels = a.channels;
        hp.n_cchunks = (a.channels + 2047) / 2048;
        hp.x = a.x;
        hp.hist = a.conv_hist;
        const long hb = (long)d.n_req * d.n_layers * hp.n_cchunks;
        if (d.op_dtype == LUMO_BF16)
            hipLaunchKernelGGL(hist_kernel<1>, dim3((unsigned)hb), dim3(256), 0, s, hp);
        else
            hipLaunchKernelGGL(hist_kernel<0>, dim3((unsigned)hb), dim3(256), 0, s, hp);
        e = hipGetLastError();
    }
    return e;
}

}  // namespace lumo
