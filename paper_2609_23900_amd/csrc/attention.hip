// Tree attention on the matrix cores (Sec. V-B; visibility Sec. III-A).
//
// Query row i (a tree node, one query head) sees its request's committed context and
// the tree nodes on its own root-to-node path. Split-K over the context, as in
// flash-decoding: a block serves (request, key/value head, 32 query nodes, one key
// range) with 2G wavefronts for G query heads that share the key/value head (up to 4
// per block; the grouped heads reuse every staged key and value tile); key ranges are the
// context partitions plus one range for the tree's own nodes. A second kernel merges
// the partial results of the ranges through their log-sum-exp.
//
// Layout per wavefront: 16 query rows of one head, one row per lane column. The
// scores are computed transposed, S^T = K Q^T (16x16x32 bf16 MFMA), so that a lane
// holds 16 scores of ONE query row (4 lane groups split the 64 keys of a tile): the
// online softmax needs only two lane-group swaps per reduction, and the probabilities
// are already in the B-operand layout of O^T = V^T P^T (key slot 8 j + e of lane group
// j is key 4 j + e of the tile's first 16-key half for e < 4, of the second for
// e >= 4). K and V tiles are staged by direct global-to-LDS copies, key-major with
// 16-byte slots XOR-swizzled by key; the V^T operand is read back with the transposing
// LDS read (ds_read_b64_tr_b16: within 16 lanes, lane i receives element i % 4 of
// lanes 4 e + i / 4, e = 0..3), so V never passes through registers. Tiles of 64 keys,
// double-buffered.
#include <mutex>

#include "device_common.h"
#include "internal.h"
#include "launch.h"

namespace lumo {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;
typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;

constexpr int kAD = 128;  // head dimension
constexpr int kAN = 32;   // query nodes per block
constexpr int kAT = 64;   // keys per tile

struct AttnParams {
    const int32_t* blob;
    int32_t o_node_off, o_row_off, o_vis, o_dfs, o_parent, o_slot;
    const int32_t* ctx_off;
    int32_t n_req, h_q, h_kv, n_split, part_len, n_nchunk, total_rows, max_nodes;
    int32_t n_hb;      // blocks per key/value head (query heads h_q / h_kv in groups of G)
    float scale_log2;  // scale * log2(e): scores in the base-2 domain
    const uint16_t* q;
    const uint16_t* k_ctx;
    const uint16_t* v_ctx;
    const uint16_t* k_tree;
    const uint16_t* v_tree;
    float* ws_o;    // [n_split + 1][total_rows][h_q][kAD]: normalised partial outputs
    float* ws_lse;  // [n_split + 1][total_rows][h_q]: partial log2-sum-exp2 (-inf: no key)
};

// max / sum over the four 16-lane rows (the same in every lane)
__device__ __forceinline__ float rows_max(float x) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    const float y = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(y), __float_as_uint(y), false, false);
    return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float rows_sum(float x) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    const float y = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(y), __float_as_uint(y), false, false);
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 w) { return __builtin_bit_cast(bf16x8, w); }

template <int G>
__global__ __launch_bounds__(128 * G, G == 1 ? 1 : 2) void attn_kernel(AttnParams p) {
    constexpr int nthr = 128 * G;
    // key and value tiles: [key][16 slots]; slot c of key t holds dims 8 (c ^ (t & 15)) .. + 7
    __shared__ uint4 kt0[kAT * 16];
    __shared__ uint4 kt1[kAT * 16];
    __shared__ uint4 vt0[kAT * 16];
    __shared__ uint4 vt1[kAT * 16];
    const int tid = (int)threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lane = tid & 63;

    int blk = xcd_remap(blockIdx.x, gridDim.x);
    const int sp = blk % (p.n_split + 1);
    blk /= p.n_split + 1;
    const int nc = blk % p.n_nchunk;
    blk /= p.n_nchunk;
    const int hb = blk % p.n_hb;
    blk /= p.n_hb;
    const int g = blk % p.h_kv;
    const int r = blk / p.h_kv;
    const int base = p.blob[p.o_node_off + r];
    const int N = p.blob[p.o_node_off + r + 1] - base;
    if (kAN * nc >= N) return;  // uniform: no query node in this chunk
    const int rbase = p.blob[p.o_row_off + r];
    const bool tree = sp == p.n_split;
    // this block's keys: tree slots [0, N), or context tokens [k0, k0 + nk)
    int k0 = 0, nk = N;
    if (!tree) {
        const int c0 = p.ctx_off[r], c1 = p.ctx_off[r + 1];
        k0 = c0 + sp * p.part_len;
        nk = max(0, min(c1 - k0, p.part_len));
    }
    const uint16_t* kmat = tree ? p.k_tree : p.k_ctx;
    const uint16_t* vmat = tree ? p.v_tree : p.v_ctx;
    const int krow0 = tree ? rbase : k0;  // absolute row of key 0 of the range

    const int h = (g * p.n_hb + hb) * G + (wave >> 1);
    const int qs = kAN * nc + 16 * (wave & 1) + (lane & 15);  // this lane's query node (slot)
    const int qrow = rbase + min(qs, N - 1);
    uint4 qf[kAD / 32];  // B operand: dims 32 ks + 8 (lane / 16) .. + 7 of the lane's query
#pragma unroll
    for (int ks = 0; ks < kAD / 32; ++ks)
        qf[ks] = *reinterpret_cast<const uint4*>(p.q + ((long)qrow * p.h_q + h) * kAD + 32 * ks + 8 * (lane >> 4));
    // tree range: the lane's query node (its preorder position gives its id), whose
    // root path is walked once per tile to mark the visible key slots
    const int qnode = tree ? p.blob[p.o_dfs + base + p.blob[p.o_vis + 2 * (base + min(qs, N - 1))]] : 0;

    const int ntile = (nk + kAT - 1) / kAT;
    // tile i of a key/value matrix into `dst`: keys past the range repeat its last key
    // (masked later, so pad rows are never read)
    auto tile_issue = [&](const uint16_t* mat, int i, uint4* dst) {
#pragma unroll
        for (int j = 0; j < kAT * 16 / nthr; ++j) {
            const int slot0 = j * nthr + 64 * wave;  // uniform
            const int slot = slot0 + lane;
            const int t = slot >> 4;
            const int kb = (slot & 15) ^ (t & 15);
            const int key = min(i * kAT + t, nk - 1);
            __builtin_amdgcn_global_load_lds(mat + ((long)(krow0 + key) * p.h_kv + g) * kAD + 8 * kb,
                                             (lds_void*)&dst[slot0], 16, 0, 0);
        }
    };

    float m = -1e30f, lsum = 0.f;  // running max (base 2) and sum of the lane's query row
    f32x4 o[kAD / 16];
#pragma unroll
    for (int dt = 0; dt < kAD / 16; ++dt)
#pragma unroll
        for (int x = 0; x < 4; ++x) o[dt][x] = 0.f;

    // visibility of the tile's 64 keys for the lane's query: a context prefix, or the
    // slots of the query's root path
    auto tile_mask = [&](int i) -> uint64_t {
        const int lo = i * kAT;
        if (!tree) {
            const int n = nk - lo;
            return n >= kAT ? ~0ull : (n <= 0 ? 0ull : ((1ull << n) - 1));
        }
        uint64_t vm = 0;
        for (int x = qnode; x >= 0; x = p.blob[p.o_parent + base + x]) {
            const int sl = p.blob[p.o_slot + base + x] - lo;
            if (sl >= 0 && sl < kAT) vm |= 1ull << sl;
        }
        return vm;
    };
    auto compute = [&](int i, const uint4* kt, const uint4* vt) {
        const uint64_t vm = tile_mask(i);
        // S^T = K Q^T: lane (query lane%16) gets keys 16 tt + 4 (lane/16) + x
        f32x4 s[kAT / 16];
#pragma unroll
        for (int tt = 0; tt < kAT / 16; ++tt) {
#pragma unroll
            for (int x = 0; x < 4; ++x) s[tt][x] = 0.f;
            const int t = 16 * tt + (lane & 15);
#pragma unroll
            for (int ks = 0; ks < kAD / 32; ++ks) {
                const bf16x8 a = as_bf16x8(kt[t * 16 + ((4 * ks + (lane >> 4)) ^ (t & 15))]);
                s[tt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, as_bf16x8(qf[ks]), s[tt], 0, 0, 0);
            }
        }
        // scale, mask, running max
        float mt = -INFINITY;
#pragma unroll
        for (int tt = 0; tt < kAT / 16; ++tt)
#pragma unroll
            for (int x = 0; x < 4; ++x) {
                const bool vis = (vm >> (16 * tt + 4 * (lane >> 4) + x)) & 1ull;
                s[tt][x] = vis ? s[tt][x] * p.scale_log2 : -INFINITY;
                mt = fmaxf(mt, s[tt][x]);
            }
        const float mn = fmaxf(m, rows_max(mt));
        const float corr = __builtin_amdgcn_exp2f(m - mn);
        m = mn;
        float ls = 0.f;
#pragma unroll
        for (int tt = 0; tt < kAT / 16; ++tt)
#pragma unroll
            for (int x = 0; x < 4; ++x) {
                s[tt][x] = __builtin_amdgcn_exp2f(s[tt][x] - mn);
                ls += s[tt][x];
            }
        lsum = lsum * corr + rows_sum(ls);
#pragma unroll
        for (int dt = 0; dt < kAD / 16; ++dt)
#pragma unroll
            for (int x = 0; x < 4; ++x) o[dt][x] *= corr;
        // O^T += V^T P^T over the two 32-key halves
#pragma unroll
        for (int kh = 0; kh < 2; ++kh) {
            const uint4 pw = make_uint4(f32x2_to_bf16x2(s[2 * kh][0], s[2 * kh][1]),
                                        f32x2_to_bf16x2(s[2 * kh][2], s[2 * kh][3]),
                                        f32x2_to_bf16x2(s[2 * kh + 1][0], s[2 * kh + 1][1]),
                                        f32x2_to_bf16x2(s[2 * kh + 1][2], s[2 * kh + 1][3]));
            // transposing reads: lane j of a 16-lane group reads dims 16 dt + 4 (j % 4) .. + 3
            // of key 32 kh + 4 (lane / 16) + j / 4 (and of that key + 16), and receives dim
            // 16 dt + j of keys 32 kh + 4 (lane / 16) + e (and + 16 + e), e = 0..3
            const int jj = lane & 15;
            const int t1 = 32 * kh + 4 * (lane >> 4) + (jj >> 2), t2 = t1 + 16;
            const char* vb = reinterpret_cast<const char*>(vt);
#pragma unroll
            for (int dt = 0; dt < kAD / 16; ++dt) {
                const int sg = 2 * dt + ((jj & 3) >> 1);  // 16-byte dim segment, then its half
                const int hb = 8 * (jj & 1);
                const v4i16 r1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (lds_v4i16*)(vb + (t1 * 16 + (sg ^ (t1 & 15))) * 16 + hb));
                const v4i16 r2 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (lds_v4i16*)(vb + (t2 * 16 + (sg ^ (t2 & 15))) * 16 + hb));
                const uint2 a1 = __builtin_bit_cast(uint2, r1), a2 = __builtin_bit_cast(uint2, r2);
                o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(make_uint4(a1.x, a1.y, a2.x, a2.y)),
                                                                as_bf16x8(pw), o[dt], 0, 0, 0);
            }
        }
    };

    if (ntile > 0) {
        tile_issue(kmat, 0, kt0);
        tile_issue(vmat, 0, vt0);
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
        for (int i = 0; i < ntile; i += 2) {
            // tile i from buffers 0 while tile i + 1 lands in buffers 1, then the reverse
            const bool n1 = i + 1 < ntile;
            if (n1) {
                tile_issue(kmat, i + 1, kt1);
                tile_issue(vmat, i + 1, vt1);
            }
            compute(i, kt0, vt0);
            if (!n1) break;
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            __syncthreads();
            const bool n2 = i + 2 < ntile;
            if (n2) {
                tile_issue(kmat, i + 2, kt0);
                tile_issue(vmat, i + 2, vt0);
            }
            compute(i + 1, kt1, vt1);
            if (!n2) break;
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            __syncthreads();
        }
    }
    if (qs >= N) return;
    // normalised partial output and its log2-sum-exp2 (-inf when no key was visible)
    const long wi = ((long)sp * p.total_rows + qrow) * p.h_q + h;
    const float inv = lsum > 0.f ? 1.f / lsum : 0.f;
#pragma unroll
    for (int dt = 0; dt < kAD / 16; ++dt)
        *reinterpret_cast<float4*>(p.ws_o + wi * kAD + 16 * dt + 4 * (lane >> 4)) =
            make_float4(o[dt][0] * inv, o[dt][1] * inv, o[dt][2] * inv, o[dt][3] * inv);
    if (lane < 16) p.ws_lse[wi] = lsum > 0.f ? m + __log2f(lsum) : -INFINITY;
}

// Merge of the key ranges of one (query row, head): weights 2^(lse_s - max). Four waves
// take every fourth range, eight ranges' loads in flight per wave, each lane two of the
// d values; the waves' sums are added in a fixed order, so the result does not depend
// on timing.
__global__ __launch_bounds__(256) void attn_combine_kernel(AttnParams p, uint16_t* __restrict__ o,
                                                           float* __restrict__ lse) {
    __shared__ float red[4];
    __shared__ float2 part[4][64];
    int blk = blockIdx.x;
    const int h = blk % p.h_q;
    blk /= p.h_q;
    const int s = blk % p.max_nodes;
    const int r = blk / p.max_nodes;
    const int N = p.blob[p.o_node_off + r + 1] - p.blob[p.o_node_off + r];
    if (s >= N) return;  // uniform over the block
    const int row = p.blob[p.o_row_off + r] + s;
    const int t = (int)threadIdx.x, lane = t & 63, wv = t >> 6;
    const int ns = p.n_split + 1;
    const long rs = (long)p.total_rows * p.h_q;  // stride between ranges
    const long ri = (long)row * p.h_q + h;
    float mx = -INFINITY;
    for (int sp = t; sp < ns; sp += 256) mx = fmaxf(mx, p.ws_lse[sp * rs + ri]);
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
    if (lane == 0) red[wv] = mx;
    __syncthreads();
    mx = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));  // finite: every node sees itself
    float wsum = 0.f, a0 = 0.f, a1 = 0.f;
    auto weight = [&](float ls) { return ls == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(ls - mx); };
    int sp = wv;
    for (; sp + 28 < ns; sp += 32) {
        float ls[8];
        float2 v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            ls[u] = p.ws_lse[(sp + 4 * u) * rs + ri];
            v[u] = *reinterpret_cast<const float2*>(p.ws_o + ((sp + 4 * u) * rs + ri) * kAD + 2 * lane);
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const float w = weight(ls[u]);
            wsum += w;
            a0 = __builtin_fmaf(w, v[u].x, a0);
            a1 = __builtin_fmaf(w, v[u].y, a1);
        }
    }
    for (; sp < ns; sp += 4) {
        const float w = weight(p.ws_lse[sp * rs + ri]);
        const float2 v = *reinterpret_cast<const float2*>(p.ws_o + (sp * rs + ri) * kAD + 2 * lane);
        wsum += w;
        a0 = __builtin_fmaf(w, v.x, a0);
        a1 = __builtin_fmaf(w, v.y, a1);
    }
    part[wv][lane] = make_float2(a0, a1);
    __syncthreads();  // also orders red[] (read above) before its reuse below
    if (lane == 0) red[wv] = wsum;
    __syncthreads();
    if (wv != 0) return;
    const float2 q0 = part[0][lane], q1 = part[1][lane], q2 = part[2][lane], q3 = part[3][lane];
    const float ws = ((red[0] + red[1]) + red[2]) + red[3];
    const float inv = 1.f / ws;
    const float b0 = ((q0.x + q1.x) + q2.x) + q3.x, b1 = ((q0.y + q1.y) + q2.y) + q3.y;
    reinterpret_cast<uint32_t*>(o + ((long)row * p.h_q + h) * kAD)[lane] = f32x2_to_bf16x2(b0 * inv, b1 * inv);
    if (lane == 0) lse[(long)row * p.h_q + h] = (mx + __log2f(ws)) * 0.69314718055994531f;
}

// Partial results of the key ranges for lumo_tree_attention_noalloc: one fixed array
// per device, held until the process ends. Host code must not pass `scratch` itself
// to a kernel (on the host it names a stand-in, not device memory); the device
// address comes from attn_scratch() below.
static __device__ __align__(256) float scratch[LUMO_TREE_ATTENTION_SCRATCH_BYTES / sizeof(float)];

}  // namespace

hipError_t attn_scratch(float** out) {
    // one lookup per device, with that device current; the address is kept per device
    constexpr int kMaxDevices = 64;
    static std::mutex mu;
    static void* addr[kMaxDevices] = {};
    *out = nullptr;
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        addr[dev] = p;
    }
    *out = static_cast<float*>(addr[dev]);
    return hipSuccess;
}

int attn_part_len(int max_ctx, int n_split) {
    const int per = (max(max_ctx, 1) + n_split - 1) / n_split;
    return (per + kAT - 1) / kAT * kAT;
}

hipError_t launch_attention(const lumo_attn_dims& d, const lumo_tree_desc& desc, const AttnArgs& a, hipStream_t s) {
    const lumo_plan& pl = desc.plan;
    if (d.n_req == 0 || pl.total_nodes == 0) return hipSuccess;
    AttnParams p;
    p.blob = desc.blob;
    p.o_node_off = pl.o_node_off;
    p.o_row_off = pl.o_row_off;
    p.o_vis = pl.o_vis;
    p.o_dfs = pl.o_dfs;
    p.o_parent = pl.o_parent;
    p.o_slot = pl.o_slot;
    p.ctx_off = a.ctx_off;
    p.n_req = d.n_req;
    p.h_q = d.h_q;
    p.h_kv = d.h_kv;
    p.n_split = a.n_split;
    p.part_len = attn_part_len(a.max_ctx, a.n_split);
    p.n_nchunk = (pl.max_nodes + kAN - 1) / kAN;
    p.total_rows = pl.total_rows;
    p.max_nodes = pl.max_nodes;
    p.scale_log2 = a.scale * 1.4426950408889634f;
    p.q = static_cast<const uint16_t*>(a.q);
    p.k_ctx = static_cast<const uint16_t*>(a.k_ctx);
    p.v_ctx = static_cast<const uint16_t*>(a.v_ctx);
    p.k_tree = static_cast<const uint16_t*>(a.k_tree);
    p.v_tree = static_cast<const uint16_t*>(a.v_tree);
    p.ws_o = a.ws;
    p.ws_lse = a.ws + (long)(a.n_split + 1) * pl.total_rows * d.h_q * kAD;
    const int grp = d.h_q / d.h_kv;
    const int gb = grp > 4 ? 4 : grp;  // query heads per block: 8 are served by two blocks
    p.n_hb = grp / gb;
    const long nb = (long)d.n_req * d.h_kv * p.n_hb * p.n_nchunk * (a.n_split + 1);
    switch (gb) {
        case 1: hipLaunchKernelGGL(attn_kernel<1>, dim3((unsigned)nb), dim3(128), 0, s, p); break;
        case 2: hipLaunchKernelGGL(attn_kernel<2>, dim3((unsigned)nb), dim3(256), 0, s, p); break;
        case 4: hipLaunchKernelGGL(attn_kernel<4>, dim3((unsigned)nb), dim3(512), 0, s, p); break;
        default: return hipErrorNotSupported;
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const long cb = (long)d.n_req * pl.max_nodes * d.h_q;
    hipLaunchKernelGGL(attn_combine_kernel, dim3((unsigned)cb), dim3(256), 0, s, p, static_cast<uint16_t*>(a.o), a.lse);
    return hipGetLastError();
}

}  // namespace lumo
