// Tree verification in WY form on the matrix cores.
//
// Unrolling Eq. (2)-(3) along a node's ancestry gives, for node t with ancestors
// a_0 (root) .. a_{d-1} and the pre-tree state R0,
//     R_t = gamma_t R0 + sum_{s ancestor-or-self of t} Gamma(s->t) delta_s k_s^T
// with gamma_t the product of alpha along root..t and Gamma(s->t) the product of
// alpha over the nodes after s up to t. Every delta then satisfies
//     delta_t = beta_t (v_t - gamma_t R0 k_t) - sum_{s strict ancestor} beta_t Gamma(s->t) (k_s.k_t) delta_s
// and the outputs are
//     o_t = gamma_t R0 q_t + sum_{s strict ancestor} Gamma(s->t) (k_s.q_t) delta_s + (k_t.q_t) delta_t.
// The only O(d^2) work per node is R0 [k_t | q_t]: a dense (d_v x d_k) x (d_k x 2N)
// contraction per instance, run on MFMA with R0 held as bf16 hi + bf16 lo (16
// significant bits) against bf16 operands (exact products, fp32 accumulation). What
// is left is a triangular system over each node's ancestors: O(N * depth) per value
// column.
//
// Two kernels:
//   coef kernel  one wavefront per (request, layer, key head). For each chunk of 32
//                nodes in depth-first preorder, an MFMA Gram block between the chunk's
//                ancestor candidates (the preorder path stack at the chunk start plus
//                the chunk itself) and the chunk's keys and queries; then per (value
//                head, node) the decay products and the coefficient record
//                {row, depth, beta, gamma, k.q, A[0..D), B[0..D)} with
//                A_m = beta Gamma(a_m->t) k_{a_m}.k_t and B_m = Gamma(a_m->t) k_{a_m}.q_t.
//   main kernel  one wavefront per (request, layer, value head, 64 value columns).
//                Loads its R0 columns once as MFMA B fragments (hi/lo bf16), computes
//                R0 k and R0 q for 32 preorder nodes at a time, exchanges half-waves
//                (permlane32 swap) so each lane owns one value column, then walks
//                the chunk in preorder keeping delta of the current path in registers
//                (the preorder path stack is exactly the ancestry).
// This replaces sequential scans; the arithmetic differs from them in rounding only
// (tolerance-level, not bitwise). The commit stays a sequential replay.
#include "device_common.h"
#include "internal.h"
#include "launch.h"

namespace lumo {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kD = 128;     // d_k = d_v
constexpr int kTile = 32;   // nodes per MFMA tile
constexpr int kStack = 16;  // ancestor candidate slots (depth index < 16)

template <int D> struct Rec {
    static constexpr int kWords = 8 + 2 * D;  // {row, depth, beta, gamma, k.q, 0, 0, 0, A[D], B[D]}
};

struct WyParams {
    const int32_t* blob;
    int32_t o_node_off, o_pre_row, o_pre_depth, o_pre_anc, o_chunk_off, o_chunk_stack, n_anc;
    int32_t n_layers, total_rows, total_nodes, h_k, h_v, group;
};

__device__ __forceinline__ bf16x8 load_bf16x8(const uint16_t* p) {
    const uint4 w = *reinterpret_cast<const uint4*>(p);
    return __builtin_bit_cast(bf16x8, w);
}

__device__ __forceinline__ bf16x8 zero_bf16x8() { return __builtin_bit_cast(bf16x8, make_uint4(0, 0, 0, 0)); }

// ------------------------------------------------------------------ coefficients
template <int D>
__global__ __launch_bounds__(64) void wy_coef_kernel(WyParams p, const uint16_t* __restrict__ kmat,
                                                     const uint16_t* __restrict__ qmat, const float* __restrict__ g,
                                                     const float* __restrict__ beta, float* __restrict__ coef) {
    constexpr int W = Rec<D>::kWords;
    __shared__ float G[2 * kTile][2 * kTile + 1];  // [candidate][chunk key | chunk query]
    int b = xcd_remap(blockIdx.x, gridDim.x);
    const int hk = b % p.h_k;
    b /= p.h_k;
    const int l = b % p.n_layers;
    const int r = b / p.n_layers;
    const int lane = threadIdx.x;
    const int base = p.blob[p.o_node_off + r];
    const int N = p.blob[p.o_node_off + r + 1] - base;
    const int32_t* prow = p.blob + p.o_pre_row + base;
    const int32_t* pdep = p.blob + p.o_pre_depth + base;
    const int32_t* panc = p.blob + p.o_pre_anc + 2L * base * p.n_anc;
    const int32_t* stack = p.blob + p.o_chunk_stack + (long)kStack * p.blob[p.o_chunk_off + r];
    const long krow0 = (long)l * p.total_rows;

    for (int c0 = 0; c0 < N; c0 += kTile, stack += kStack) {
        // Gram candidates: slots 0..15 the chunk's path stack, 16..47 the chunk itself
        int cand[2];
#pragma unroll
        for (int mt = 0; mt < 2; ++mt) {
            const int ci = mt * kTile + lane % kTile;
            int rw = -1;
            if (ci < kStack) {
                rw = stack[ci];
            } else if (ci < kStack + kTile) {
                const int pos = c0 + ci - kStack;
                if (pos < N) rw = prow[pos];
            }
            cand[mt] = rw;
        }
        const int tpos = c0 + lane % kTile;
        const int trow = tpos < N ? prow[tpos] : -1;
        f32x16 acc[2][2];
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
#pragma unroll
            for (int ct = 0; ct < 2; ++ct)
#pragma unroll
                for (int e = 0; e < 16; ++e) acc[mt][ct][e] = 0.f;
#pragma unroll
        for (int s = 0; s < kD / 16; ++s) {
            const int kk = 16 * s + 8 * (lane / kTile);
            bf16x8 a[2];
#pragma unroll
            for (int mt = 0; mt < 2; ++mt)
                a[mt] = cand[mt] >= 0 ? load_bf16x8(kmat + ((krow0 + cand[mt]) * p.h_k + hk) * kD + kk) : zero_bf16x8();
            const bf16x8 bk = trow >= 0 ? load_bf16x8(kmat + ((krow0 + trow) * p.h_k + hk) * kD + kk) : zero_bf16x8();
            const bf16x8 bq = trow >= 0 ? load_bf16x8(qmat + ((krow0 + trow) * p.h_k + hk) * kD + kk) : zero_bf16x8();
#pragma unroll
            for (int mt = 0; mt < 2; ++mt) {
                acc[mt][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[mt], bk, acc[mt][0], 0, 0, 0);
                acc[mt][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[mt], bq, acc[mt][1], 0, 0, 0);
            }
        }
        // MFMA 32x32 output: lane holds column lane%32, rows 8(e/4) + 4(lane/32) + e%4
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
#pragma unroll
            for (int ct = 0; ct < 2; ++ct)
#pragma unroll
                for (int e = 0; e < 16; ++e)
                    G[mt * kTile + 8 * (e / 4) + 4 * (lane / kTile) + e % 4][ct * kTile + lane % kTile] = acc[mt][ct][e];
        __syncthreads();

        const int t = lane % kTile;
        const int pos = c0 + t;
        if (pos < N) {
            const int d = pdep[pos];
            const int rn = prow[pos];
            int ci[D], arow[D];
#pragma unroll
            for (int m = 0; m < D; ++m) {
                ci[m] = m < d ? panc[2 * ((long)pos * p.n_anc + m)] : 0;
                arow[m] = m < d ? panc[2 * ((long)pos * p.n_anc + m) + 1] : rn;
            }
            for (int hv = hk * p.group + lane / kTile; hv < (hk + 1) * p.group; hv += 2) {
                float* out = coef + (((long)l * p.h_v + hv) * p.total_nodes + base + pos) * W;
                const long gi = (krow0 + rn) * p.h_v + hv;
                const float bn = beta[gi];
                float al[D];
#pragma unroll
                for (int m = 0; m < D; ++m) al[m] = __expf(g[(krow0 + arow[m]) * p.h_v + hv]);
                // Gamma(a_m -> n) = product of alpha over the ancestors deeper than m and n
                float gam = __expf(g[gi]);
#pragma unroll
                for (int m = D - 1; m >= 0; --m) {
                    const bool live = m < d;
                    out[8 + m] = live ? bn * gam * G[ci[m]][t] : 0.f;
                    out[8 + D + m] = live ? gam * G[ci[m]][kTile + t] : 0.f;
                    if (live) gam *= al[m];
                }
                out[0] = __int_as_float(rn);
                out[1] = __int_as_float(d);
                out[2] = bn;
                out[3] = gam;  // gamma_n: product of alpha over root..n
                out[4] = G[kStack + t][kTile + t];  // k_n . q_n
                out[5] = 0.f;
                out[6] = 0.f;
                out[7] = 0.f;
            }
        }
        __syncthreads();
    }
}

// ------------------------------------------------------------------ main kernel
// Staging of one chunk (32 preorder nodes) into LDS: the chunk's coefficient records
// (a contiguous block of the table) and its value rows restricted to this wave's 64
// columns. Copied with direct global-to-LDS loads (no registers), one chunk ahead,
// so the per-node recursion reads only LDS and registers.
template <int D>
struct Stage {
    static constexpr int W = Rec<D>::kWords;
    static constexpr int kRec4 = kTile * W / 4;  // float4 slots, a multiple of 64
    static_assert(kRec4 % 64 == 0, "record block must tile the wave");
    float4 rec[kRec4];
    uint4 v[kTile * 8];  // [node][8 segments of 8 bf16]
};

typedef __attribute__((address_space(3))) void lds_void;

template <int D>
__device__ __forceinline__ void stage_issue(Stage<D>& st, const float* __restrict__ cbase,
                                            const uint16_t* __restrict__ vmat, int c0, int nv, int myrow,
                                            long krow0, int h_v, int h, int j0, int lane) {
    constexpr int W4 = Rec<D>::kWords / 4;
    // lane i of round k copies float4 (64 k + i) to LDS slot 64 k + i; the record slots
    // of nodes past the chunk's end receive copies of its last record.
    const float4* src = reinterpret_cast<const float4*>(cbase + (long)c0 * W4 * 4);
#pragma unroll
    for (int k = 0; k < Stage<D>::kRec4 / 64; ++k) {
        const int i = 64 * k + lane;
        const int n = i / W4;
        __builtin_amdgcn_global_load_lds(src + (n < nv ? i : (nv - 1) * W4 + i % W4), (lds_void*)&st.rec[64 * k], 16,
                                         0, 0);
    }
    // value rows: slot p = 64 k + lane holds node p / 8, columns j0 + 8 (p % 8) .. + 7;
    // myrow of lane n is the row of node n (the last node's row past the end)
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int pidx = 64 * k + lane;
        const int n = pidx >> 3;
        const int rn = __shfl(myrow, n);
        const uint16_t* g = vmat + ((krow0 + rn) * h_v + h) * kD + j0 + 8 * (pidx & 7);
        __builtin_amdgcn_global_load_lds(g, (lds_void*)&st.v[64 * k], 16, 0, 0);
    }
}

// Key and query rows of a chunk, staged once per block and shared by its waves:
// [key | query][32 nodes][16 slots of 8 bf16]; key block kb of node n sits in slot
// kb ^ (n & 15), so the fragment reads of a half-wave (32 nodes, one key block)
// spread over all banks.
struct KQTile {
    uint4 slot[2 * kTile * 16];
};

constexpr int kMaxWaves = 4;  // 2 value heads x 2 column halves per block

template <int D>
constexpr size_t wy_lds_bytes() {
    return sizeof(KQTile) + kMaxWaves * 2 * sizeof(Stage<D>);
}

template <int D, int NVH>
__global__ __launch_bounds__(256, 2) void wy_main_kernel(WyParams p, const uint16_t* __restrict__ kmat,
                                                         const uint16_t* __restrict__ qmat,
                                                         const uint16_t* __restrict__ vmat,
                                                         const float* __restrict__ state0,
                                                         const float* __restrict__ coef, uint16_t* __restrict__ out) {
    constexpr int W = Rec<D>::kWords;
    extern __shared__ uint4 lds[];
    KQTile& tile = *reinterpret_cast<KQTile*>(lds);
    constexpr int nthr = 128 * NVH;           // NVH value heads x 2 column halves per block
    const int tid = (int)threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: head and half in SGPRs
    const int lane = tid & 63;
    Stage<D>* stage = reinterpret_cast<Stage<D>*>(lds + sizeof(KQTile) / 16) + 2 * wave;

    int b = xcd_remap(blockIdx.x, gridDim.x);
    const int pairs = p.group / NVH;
    const int pp = b % pairs;
    b /= pairs;
    const int hk = b % p.h_k;
    b /= p.h_k;
    const int l = b % p.n_layers;
    const int r = b / p.n_layers;
    const int h = hk * p.group + pp * NVH + (wave >> 1);
    const int half = wave & 1;
    const int j0 = 64 * half;
    const int base = p.blob[p.o_node_off + r];
    const int N = p.blob[p.o_node_off + r + 1] - base;
    if (N <= 0) return;  // uniform over the block
    const int32_t* prow = p.blob + p.o_pre_row + base;
    const long krow0 = (long)l * p.total_rows;
    const float* cbase = coef + (((long)l * p.h_v + h) * p.total_nodes + base) * W;

    // rows feeding this thread's tile slots (slot g = round * nthr + tid) for chunk c0
    constexpr int rounds = 2 * kTile * 16 / nthr;  // 4 or 8
    auto tile_rows = [&](int c0, int (&rows)[rounds]) {
#pragma unroll
        for (int j = 0; j < rounds; ++j) {
            const int n = ((j * nthr + tid) >> 4) & (kTile - 1);
            const int pos = c0 + n;
            rows[j] = prow[pos < N ? pos : N - 1];
        }
    };
    auto tile_issue = [&](const int (&rows)[rounds]) {
#pragma unroll
        for (int j = 0; j < rounds; ++j) {
            const int g = j * nthr + tid;
            const int n = (g >> 4) & (kTile - 1);
            const int kb = (g & 15) ^ (n & 15);
            const uint16_t* src = (g >= kTile * 16 ? qmat : kmat) + ((krow0 + rows[j]) * p.h_k + hk) * kD + 8 * kb;
            __builtin_amdgcn_global_load_lds(src, (lds_void*)&tile.slot[j * nthr + 64 * wave], 16, 0, 0);
        }
    };
    auto node_row = [&](int c0) {
        const int pos = c0 + lane % kTile;
        return prow[pos < N ? pos : N - 1];
    };

    int trows[rounds];
    tile_rows(0, trows);
    tile_issue(trows);
    int vrow = node_row(0);
    stage_issue<D>(stage[0], cbase, vmat, 0, min(kTile, N), vrow, krow0, p.h_v, h, j0, lane);

    // R0 columns j0 + 32 ct + lane%32 as MFMA B fragments: keys 16 s + 8 (lane/32) + e.
    const float* S = state0 + (((long)r * p.n_layers + l) * p.h_v + h) * (long)(kD * kD);
    const float* Sl = S + (long)(8 * (lane / kTile)) * kD + j0 + lane % kTile;
    bf16x8 bhi[2][kD / 16], blo[2][kD / 16];
    // Each fp32 value x is held as hi + lo: hi = x truncated to bf16, lo = the exact
    // remainder x - hi rounded to nearest bf16 (|x - hi - lo| <= 2^-15 |x|).
#pragma unroll
    for (int ct = 0; ct < 2; ++ct)
#pragma unroll
        for (int s = 0; s < kD / 16; ++s) {
            uint32_t hw[4], lw[4];
#pragma unroll
            for (int e2 = 0; e2 < 4; ++e2) {
                const uint32_t x0 = __float_as_uint(Sl[(long)(16 * s + 2 * e2) * kD + kTile * ct]);
                const uint32_t x1 = __float_as_uint(Sl[(long)(16 * s + 2 * e2 + 1) * kD + kTile * ct]);
                hw[e2] = __builtin_amdgcn_perm(x1, x0, 0x07060302u);  // {hi(x1), hi(x0)}: upper halves
                lw[e2] = f32x2_to_bf16x2(__uint_as_float(x0) - __uint_as_float(x0 & 0xffff0000u),
                                         __uint_as_float(x1) - __uint_as_float(x1 & 0xffff0000u));
            }
            bhi[ct][s] = __builtin_bit_cast(bf16x8, make_uint4(hw[0], hw[1], hw[2], hw[3]));
            blo[ct][s] = __builtin_bit_cast(bf16x8, make_uint4(lw[0], lw[1], lw[2], lw[3]));
        }

    // delta of the current path by depth; slot D takes the writes of nodes at depth D,
    // which have no descendants (their delta is never read)
    float dst[D + 1];
#pragma unroll
    for (int m = 0; m <= D; ++m) dst[m] = 0.f;
    const int vcol = j0 + lane;
    const int n_a = lane % kTile;               // node of this lane's A fragment rows
    const int kb0 = lane / kTile;               // key block offset within a 16-key step

    for (int c0 = 0, buf = 0; c0 < N; c0 += kTile, buf ^= 1) {
        const bool more = c0 + kTile < N;
        if (more) {  // rows of the next chunk, needed once this chunk's tile is consumed
            tile_rows(c0 + kTile, trows);
            vrow = node_row(c0 + kTile);
        }
        // this chunk's tile and staging have landed for every wave of the block
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
        // the other staging buffer was last read by the previous chunk's recursion
        if (more)
            stage_issue<D>(stage[buf ^ 1], cbase, vmat, c0 + kTile, min(kTile, N - c0 - kTile), vrow, krow0,
                           p.h_v, h, j0, lane);
        f32x16 ak[2], aq[2];
#pragma unroll
        for (int ct = 0; ct < 2; ++ct)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                ak[ct][e] = 0.f;
                aq[ct][e] = 0.f;
            }
#pragma unroll
        for (int s = 0; s < kD / 16; ++s) {
            const int kb = 2 * s + kb0;
            const bf16x8 fk = __builtin_bit_cast(bf16x8, tile.slot[n_a * 16 + (kb ^ (n_a & 15))]);
            const bf16x8 fq = __builtin_bit_cast(bf16x8, tile.slot[(kTile + n_a) * 16 + (kb ^ (n_a & 15))]);
#pragma unroll
            for (int ct = 0; ct < 2; ++ct) {
                ak[ct] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fk, bhi[ct][s], ak[ct], 0, 0, 0);
                ak[ct] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fk, blo[ct][s], ak[ct], 0, 0, 0);
                aq[ct] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fq, bhi[ct][s], aq[ct], 0, 0, 0);
                aq[ct] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fq, blo[ct][s], aq[ct], 0, 0, 0);
            }
        }
        __syncthreads();  // every wave has read the tile: it may be refilled
        if (more) tile_issue(trows);
        // Lane l holds column 32 ct + l%32 of tile ct for nodes 8(e/4) + 4(l/32) + e%4.
        // Swapping tile 0's upper half-wave with tile 1's lower half-wave leaves every
        // lane with one column (j0 + lane): [0][e] = node 8(e/4) + e%4, [1][e] = node 8(e/4) + 4 + e%4.
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            const auto sk = __builtin_amdgcn_permlane32_swap(__float_as_uint(ak[0][e]), __float_as_uint(ak[1][e]), false, false);
            ak[0][e] = __uint_as_float(sk[0]);
            ak[1][e] = __uint_as_float(sk[1]);
            const auto sq = __builtin_amdgcn_permlane32_swap(__float_as_uint(aq[0][e]), __float_as_uint(aq[1][e]), false, false);
            aq[0][e] = __uint_as_float(sq[0]);
            aq[1][e] = __uint_as_float(sq[1]);
        }
        const float* rec = reinterpret_cast<const float*>(stage[buf].rec);
        const uint16_t* vs = reinterpret_cast<const uint16_t*>(stage[buf].v);
        // Straight-line over all 32 slots: slots past the chunk's end hold exact copies of
        // its last node (tile rows, value row, record), so they recompute that node's
        // delta and output bit for bit and store the same value to the same place.
#pragma unroll
        for (int n = 0; n < kTile; ++n) {
            const int e = 4 * (n / 8) + n % 4;
            const float pk = ((n / 4) & 1) ? ak[1][e] : ak[0][e];
            const float pq = ((n / 4) & 1) ? aq[1][e] : aq[0][e];
            const float* cf = rec + n * W;
            const int rn = __builtin_amdgcn_readfirstlane(__float_as_int(cf[0]));  // uniform
            const int d = __builtin_amdgcn_readfirstlane(__float_as_int(cf[1]));
            const float bn = cf[2], gm = cf[3], cn = cf[4];
            const float vj = __uint_as_float(((uint32_t)vs[n * 64 + lane]) << 16);
            float sa = 0.f, sb = 0.f;
#pragma unroll
            for (int m = 0; m < D; ++m) {
                sa = __builtin_fmaf(cf[8 + m], dst[m], sa);
                sb = __builtin_fmaf(cf[8 + D + m], dst[m], sb);
            }
            const float u = __builtin_fmaf(-gm, pk, vj);           // v - gamma R0 k
            const float delta = __builtin_fmaf(bn, u, -sa);        // beta u - sum A delta
            const float ov = __builtin_fmaf(cn, delta, __builtin_fmaf(gm, pq, sb));
            dst[d < D ? d : D] = delta;  // uniform index: an indexed register write
            uint16_t* orow = out + ((krow0 + rn) * p.h_v + h) * kD;
            orow[vcol] = f32_to_bf16(ov);
        }
    }
}

template <int D, int NVH>
hipError_t launch_wy_main(const lumo_gdn_dims& d, const WyParams& p, const uint16_t* k, const uint16_t* q,
                          const uint16_t* v, const GdnArgs& a, hipStream_t s) {
    const long mb = (long)d.n_req * d.n_layers * d.h_k * (p.group / NVH);
    static bool attr_set = false;  // LDS above the 64 KB default (same value for every call)
    if (!attr_set) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&wy_main_kernel<D, NVH>),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)wy_lds_bytes<D>());
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    hipLaunchKernelGGL((wy_main_kernel<D, NVH>), dim3((unsigned)mb), dim3(128 * NVH), wy_lds_bytes<D>(), s, p, k, q,
                       v, a.state0, a.ws, static_cast<uint16_t*>(a.o));
    return hipGetLastError();
}

template <int D>
hipError_t launch_wy_d(const lumo_gdn_dims& d, const lumo_tree_desc& desc, const GdnArgs& a, hipStream_t s) {
    const lumo_plan& pl = desc.plan;
    WyParams p;
    p.blob = desc.blob;
    p.o_node_off = pl.o_node_off;
    p.o_pre_row = pl.o_pre_row;
    p.o_pre_depth = pl.o_pre_depth;
    p.o_pre_anc = pl.o_pre_anc;
    p.o_chunk_off = pl.o_chunk_off;
    p.o_chunk_stack = pl.o_chunk_stack;
    p.n_anc = pl.n_anc;
    p.n_layers = d.n_layers;
    p.total_rows = pl.total_rows;
    p.total_nodes = pl.total_nodes;
    p.h_k = d.h_k;
    p.h_v = d.h_v;
    p.group = d.h_v / d.h_k;
    const auto* k = static_cast<const uint16_t*>(a.k);
    const auto* q = static_cast<const uint16_t*>(a.q);
    const auto* v = static_cast<const uint16_t*>(a.v);
    const long cb = (long)d.n_req * d.n_layers * d.h_k;
    hipLaunchKernelGGL(wy_coef_kernel<D>, dim3((unsigned)cb), dim3(64), 0, s, p, k, q, a.g, a.beta, a.ws);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    // one block per (request, layer, key head, pair of value heads): the pair's
    // waves share the staged key and query rows
    if (p.group % 2 == 0)
        return launch_wy_main<D, 2>(d, p, k, q, v, a, s);
    return launch_wy_main<D, 1>(d, p, k, q, v, a, s);
}

}  // namespace

int wy_stack_depth(const lumo_plan& pl) { return pl.max_depth <= 9 ? 8 : 16; }

size_t wy_workspace_bytes(const lumo_gdn_dims& d, const lumo_plan& pl) {
    const int D = wy_stack_depth(pl);
    return (size_t)pl.total_nodes * d.n_layers * d.h_v * (8 + 2 * D) * sizeof(float);
}

hipError_t launch_wy(const lumo_gdn_dims& d, const lumo_tree_desc& desc, const GdnArgs& a, hipStream_t s) {
    if (desc.plan.max_depth > kStack + 1) return hipErrorNotSupported;
    return wy_stack_depth(desc.plan) == 8 ? launch_wy_d<8>(d, desc, a, s) : launch_wy_d<16>(d, desc, a, s);
}

}  // namespace lumo
