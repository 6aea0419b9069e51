// Tree verification in WY form on the vector ALUs: the shapes the matrix-core kernel
// (verify_wy.hip) does not take -- fp32 operands, d_k or d_v below 128, and paths of up
// to kWyvMaxDepth nodes -- with the same arithmetic form and no cut states.
//
// Unrolling Eq. (2)-(3) along a node's ancestry a_0 (root) .. a_{d-1}, t:
//     R_t = gamma_t R0 + sum_{s ancestor-or-self of t} Gamma(s->t) delta_s k_s^T
//     delta_t = beta_t (v_t - gamma_t R0 k_t) - sum_m A_m delta_{a_m},
//         A_m = beta_t Gamma(a_m->t) (k_{a_m} . k_t)
//     o_t = gamma_t R0 q_t + sum_m B_m delta_{a_m} + (k_t . q_t) delta_t,
//         B_m = Gamma(a_m->t) (k_{a_m} . q_t)
// with gamma_t the product of alpha along root..t and Gamma(a_m->t) the product over the
// nodes after a_m up to t (products, never ratios). With query/key normalisation
// (Sec. IV-B) every key and query enters through its factor 1/sqrt(|x|^2 + eps).
//
// A block serves (request, layer, key head) and up to four wavefronts of that key
// head's (value head, 64-column tile) pairs, and walks the request's nodes in
// depth-first preorder, one node at a time:
//   1. the node's key and query rows go to LDS as fp32; the key row is kept by depth,
//      so the rows of the current root path are the node's ancestors;
//   2. the block forms the node's Gram entries k_{a_m}.k_t, k_{a_m}.q_t, k_t.q_t and the
//      squared norms (8 to 16 lanes per dot product);
//   3. each wavefront (one value head, 64 value columns) holds its columns of R0 in
//      registers for the whole walk, a lane a quarter of the keys of four columns; it
//      takes R0 k_t and R0 q_t against the LDS rows (each lane reads a quarter of each
//      row, and the four quarters' sums are added across lanes), after which a lane
//      serves one column: the decays of the path from its LDS stack, the coefficients
//      (lane m forms A_m and B_m by a suffix product over the lanes), and the deltas of
//      its column by depth from LDS.
// The state is read once per wavefront and nothing is written besides the outputs.
#include "device_common.h"
#include "internal.h"
#include "launch.h"

namespace lumo {
namespace {

constexpr int kWpb = 4;  // wavefronts per block

struct WyvParams {
    const int32_t* blob;
    int32_t o_node_off, o_pre_row, o_pre_depth;
    int32_t n_layers, total_rows, h_k, h_v, d_v, group, n_vt, nwk, n_wb, max_depth;
    int32_t qkn, raw_gates;
    float qk_eps;
    const float* a_log;
    const float* dt_bias;
};

// LDS layout (floats), for max_depth Dm and key dimension DK:
//   kst   [Dm][DK + 4]  key rows of the current root path by depth (row d: the node)
//   cq    [DK]          the node's query row
//   gram  [2 Dm + 4]    k_{a_m}.k_t (m < Dm), k_{a_m}.q_t, then k.q, |k|^2, |q|^2
//   knrm  [Dm]          1/sqrt(|k|^2 + eps) of the path's keys (normalisation)
//   per wave: ast [Dm] decays of the path (then 2 Dm unused),
//             dst [Dm][64] deltas of the path, one column per lane
template <int DK> struct WyvLds {
    int Dm;
    __device__ __host__ int kst() const { return 0; }
    __device__ __host__ int cq() const { return Dm * (DK + 4); }
    __device__ __host__ int gram() const { return cq() + DK; }
    __device__ __host__ int knrm() const { return gram() + 2 * Dm + 4; }
    __device__ __host__ int wave0() const { return knrm() + Dm; }
    __device__ __host__ int wave_floats() const { return 3 * Dm + 64 * Dm; }
    __device__ __host__ int total() const { return wave0() + kWpb * wave_floats(); }
};

template <int DK, int OPT>
__global__ __launch_bounds__(256) void wyv_kernel(WyvParams p, const int32_t* __restrict__ blob,
                                                  const typename Op<OPT>::T* __restrict__ q,
                                                  const typename Op<OPT>::T* __restrict__ k,
                                                  const typename Op<OPT>::T* __restrict__ v,
                                                  const float* __restrict__ g, const float* __restrict__ gbeta,
                                                  const float* __restrict__ state0, typename Op<OPT>::T* __restrict__ o) {
    using T = typename Op<OPT>::T;
    extern __shared__ __attribute__((aligned(16))) float lds[];
    static_assert(DK % 16 == 0 && DK <= 128, "key dimension");
    constexpr int kG = DK >= 64 ? 16 : DK / 8;  // lanes per Gram dot product
    constexpr int kE = DK / kG;                 // elements per lane (8)
    constexpr int kPer = 16 / (int)sizeof(T);   // row elements per 16-byte piece
    constexpr int kPieces = DK / kPer;          // pieces per row
    static_assert(2 * kPieces <= 64, "one piece of the key and query rows per thread of a wave");
    const WyvLds<DK> L{p.max_depth};
    float* kst = lds + L.kst();
    float* cq = lds + L.cq();
    float* gram = lds + L.gram();
    float* knrm = lds + L.knrm();
    const int Dm = p.max_depth;

    const int tid = (int)threadIdx.x;
    const int nthr = (int)blockDim.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lane = tid & 63;
    float* ast = lds + L.wave0() + wave * L.wave_floats();
    float* dst = ast + 3 * Dm;  // [Dm][64]

    int blk = xcd_remap(blockIdx.x, gridDim.x);
    const int wb = blk % p.n_wb;
    blk /= p.n_wb;
    const int hk = blk % p.h_k;
    blk /= p.h_k;
    const int l = blk % p.n_layers;
    const int r = blk / p.n_layers;
    const int base = blob[p.o_node_off + r];
    const int N = blob[p.o_node_off + r + 1] - base;
    if (N <= 0) return;  // uniform over the block
    const int gw = wb * kWpb + wave;  // this wave's (value head, column tile) of the key head
    const bool wact = gw < p.nwk;     // uniform: idle waves take part in the barriers only
    const int h = hk * p.group + (wact ? gw / p.n_vt : 0);
    // R0 fragment of a lane: keys kg KQ .. kg KQ + KQ - 1 (kg = lane / 16) of the 4 adjacent
    // columns j0 + 4 cg .. + 3 (cg = lane % 16); after the products the lane serves
    // column j0 + 4 cg + kg
    constexpr int KQ = DK / 4;
    const int cg = lane % 16, kg = lane / 16;
    const int j0 = (wact ? gw % p.n_vt : 0) * 64;
    const int j = j0 + 4 * cg + kg;
    const bool cact = wact && j < p.d_v;
    const int jc = j < p.d_v ? j : p.d_v - 1;
    const int cgc = j0 + 4 * cg + 4 <= p.d_v ? cg : (p.d_v - j0) / 4 - 1;  // a valid group to read
    const bool qkn = p.qkn != 0;
    const bool rawg = p.raw_gates != 0;
    const float alog = rawg ? p.a_log[l * p.h_v + h] : 0.f;
    const float dtb = rawg ? p.dt_bias[l * p.h_v + h] : 0.f;
    const long lrow = (long)l * p.total_rows;
    const int32_t* prow = blob + p.o_pre_row + base;
    const int32_t* pdep = blob + p.o_pre_depth + base;

    // the wave's columns of the pre-tree state, for the whole walk: rf[i] holds key
    // kg KQ + i of the lane's four columns (one 16-byte load per key)
    float4 rf[KQ];
    {
        const float* S = state0 + (((long)r * p.n_layers + l) * p.h_v + h) * (long)DK * p.d_v + j0 + 4 * cgc;
#pragma unroll
        for (int i = 0; i < KQ; ++i) rf[i] = *reinterpret_cast<const float4*>(S + (long)(kg * KQ + i) * p.d_v);
    }

    // Thread tid < 2 kPieces of the block carries piece tid of a node's [key | query]
    // row (16 bytes); the others load a valid piece that is not used.
    const int pc = tid < 2 * kPieces ? tid : 0;
    const bool pown = tid < 2 * kPieces;
    auto piece = [&](int row) -> uint4 {
        const T* src = (pc < kPieces ? k : q) + ((lrow + row) * p.h_k + hk) * DK + (pc % kPieces) * kPer;
        return *reinterpret_cast<const uint4*>(src);
    };
    int row = prow[0];
    int dep = pdep[0];
    uint4 xp = piece(row);
    float vj = Op<OPT>::ld(v, ((lrow + row) * p.h_v + h) * p.d_v + jc);
    float gv = g[(lrow + row) * p.h_v + h], bv = gbeta[(lrow + row) * p.h_v + h];

    for (int pos = 0; pos < N; ++pos) {
        const int d = dep;  // uniform
        const int rw = row;
        const float vt = vj, gt = gv, bt = bv;
        // ---- 1. the node's rows into LDS as fp32 (the key row at depth d)
        __syncthreads();  // every wave is done with the previous node's rows
        if (pown) {
            float* dstp = pc < kPieces ? kst + d * (DK + 4) + pc * kPer : cq + (pc - kPieces) * kPer;
            if constexpr (OPT == 1) {
                *reinterpret_cast<float4*>(dstp) = make_float4(bf16_lo(xp.x), bf16_hi(xp.x), bf16_lo(xp.y), bf16_hi(xp.y));
                *reinterpret_cast<float4*>(dstp + 4) =
                    make_float4(bf16_lo(xp.z), bf16_hi(xp.z), bf16_lo(xp.w), bf16_hi(xp.w));
            } else {
                *reinterpret_cast<uint4*>(dstp) = xp;
            }
        }
        if (pos + 1 < N) {  // the next node's operands, in flight during this node
            row = prow[pos + 1];
            dep = pdep[pos + 1];
            xp = piece(row);
            vj = Op<OPT>::ld(v, ((lrow + row) * p.h_v + h) * p.d_v + jc);
            gv = g[(lrow + row) * p.h_v + h];
            bv = gbeta[(lrow + row) * p.h_v + h];
        }
        __syncthreads();
        // ---- 2. Gram entries: dot e < d: k_{a_e}.k_t; d <= e < 2d: k_{a_{e-d}}.q_t;
        // 2d: k_t.q_t; 2d + 1: |k_t|^2; 2d + 2: |q_t|^2
        const int nd = 2 * d + 3;
        const float* kt = kst + d * (DK + 4);
        for (int e0 = 0; e0 < nd; e0 += nthr / kG) {
            const int e = e0 + tid / kG;
            const int part = tid % kG;
            const int ea = e < 2 * d ? (e < d ? e : e - d) : d;  // row of the first operand
            const float* xa = e == 2 * d + 2 ? cq : kst + ea * (DK + 4);
            const float* xb = (e < d || e == 2 * d + 1) ? kt : cq;
            float s0 = 0.f, s1 = 0.f;
#pragma unroll
            for (int i = 0; i < kE; i += 4) {
                const float4 a4 = *reinterpret_cast<const float4*>(xa + part * kE + i);
                const float4 b4 = *reinterpret_cast<const float4*>(xb + part * kE + i);
                s0 = __builtin_fmaf(a4.x, b4.x, s0);
                s1 = __builtin_fmaf(a4.y, b4.y, s1);
                s0 = __builtin_fmaf(a4.z, b4.z, s0);
                s1 = __builtin_fmaf(a4.w, b4.w, s1);
            }
            float s = s0 + s1;
#pragma unroll
            for (int off = kG / 2; off >= 1; off >>= 1) s += __shfl_xor(s, off);
            if (e < nd && part == 0) gram[e < 2 * d ? (e < d ? e : Dm + (e - d)) : 2 * Dm + (e - 2 * d)] = s;
        }
        __syncthreads();
        if (!wact) continue;
        // ---- 3. this wave's head and columns
        const float nk = qkn ? __builtin_amdgcn_rsqf(gram[2 * Dm + 1] + p.qk_eps) : 1.f;
        const float nq = qkn ? __builtin_amdgcn_rsqf(gram[2 * Dm + 2] + p.qk_eps) : 1.f;
        const float alpha = __expf(rawg ? raw_log_alpha(gt, alog, dtb) : gt);
        const float beta = rawg ? raw_beta(bt) : bt;
        // coefficients: lane m < d forms A_m and B_m. Gamma(a_m -> t) = alpha_t times the
        // product of the decays at depths m+1 .. d-1: a suffix product over the lanes
        // (lane m reads the decay at depth m; lanes past the path hold 1).
        float sp = lane < d ? ast[lane] : 1.f;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const float t = __shfl_down(sp, off);
            sp = lane + off < 64 ? sp * t : sp;
        }
        const float nxt = __shfl_down(sp, 1);
        const float gm = alpha * (lane + 1 < 64 ? nxt : 1.f);  // Gamma(a_lane -> t)
        const float gam = alpha * __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(sp)));  // gamma_t
        const float nkm = (qkn && lane < d) ? knrm[lane] : 1.f;
        const float cA = beta * gm * (gram[lane < d ? lane : 0] * (nkm * nk));
        const float cB = gm * (gram[Dm + (lane < d ? lane : 0)] * (nkm * nq));
        // R0 k_t and R0 q_t: each lane takes its KQ keys of the four columns against the
        // rows in LDS (lanes of a key group read the same addresses), the four key groups'
        // partial sums are added across the lane rows, and the lane keeps its column's
        float u0, w0;
        {
            float su[4] = {0.f, 0.f, 0.f, 0.f}, sw[4] = {0.f, 0.f, 0.f, 0.f};
            const float* kr = kt + kg * KQ;
            const float* qr = cq + kg * KQ;
#pragma unroll
            for (int i = 0; i < KQ; i += 4) {
                const float4 k4 = *reinterpret_cast<const float4*>(kr + i);
                const float4 q4 = *reinterpret_cast<const float4*>(qr + i);
                const float kv[4] = {k4.x, k4.y, k4.z, k4.w}, qv[4] = {q4.x, q4.y, q4.z, q4.w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float4 f = rf[i + e];
                    su[0] = __builtin_fmaf(f.x, kv[e], su[0]);
                    su[1] = __builtin_fmaf(f.y, kv[e], su[1]);
                    su[2] = __builtin_fmaf(f.z, kv[e], su[2]);
                    su[3] = __builtin_fmaf(f.w, kv[e], su[3]);
                    sw[0] = __builtin_fmaf(f.x, qv[e], sw[0]);
                    sw[1] = __builtin_fmaf(f.y, qv[e], sw[1]);
                    sw[2] = __builtin_fmaf(f.z, qv[e], sw[2]);
                    sw[3] = __builtin_fmaf(f.w, qv[e], sw[3]);
                }
            }
            float uc[4], wc[4];
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                uc[c] = row_group_sum(su[c]);
                wc[c] = row_group_sum(sw[c]);
            }
            u0 = kg == 0 ? uc[0] : kg == 1 ? uc[1] : kg == 2 ? uc[2] : uc[3];
            w0 = kg == 0 ? wc[0] : kg == 1 ? wc[1] : kg == 2 ? wc[2] : wc[3];
        }
        // sums over the path's deltas: the coefficients from lane m, the delta of the
        // lane's column at depth m from LDS (even and odd depths apart)
        float sa0 = 0.f, sa1 = 0.f, sb0 = 0.f, sb1 = 0.f;
        int m = 0;
        for (; m + 1 < d; m += 2) {
            const float d0 = dst[m * 64 + lane], d1 = dst[(m + 1) * 64 + lane];
            const float a0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(cA), m));
            const float b0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(cB), m));
            const float a1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(cA), m + 1));
            const float b1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(cB), m + 1));
            sa0 = __builtin_fmaf(a0, d0, sa0);
            sb0 = __builtin_fmaf(b0, d0, sb0);
            sa1 = __builtin_fmaf(a1, d1, sa1);
            sb1 = __builtin_fmaf(b1, d1, sb1);
        }
        if (m < d) {
            const float d0 = dst[m * 64 + lane];
            sa0 = __builtin_fmaf(__int_as_float(__builtin_amdgcn_readlane(__float_as_int(cA), m)), d0, sa0);
            sb0 = __builtin_fmaf(__int_as_float(__builtin_amdgcn_readlane(__float_as_int(cB), m)), d0, sb0);
        }
        const float delta = __builtin_fmaf(beta, __builtin_fmaf(-(gam * nk), u0, vt), -(sa0 + sa1));
        const float ov = __builtin_fmaf(gram[2 * Dm] * (nk * nq), delta, __builtin_fmaf(gam * nq, w0, sb0 + sb1));
        dst[d * 64 + lane] = delta;
        if (lane == 0) {
            ast[d] = alpha;
            if (wave == 0) knrm[d] = nk;  // one writer; read by later nodes only
        }
        if (cact) Op<OPT>::st(o, ((lrow + rw) * p.h_v + h) * (long)p.d_v + j, ov);
    }
}

template <int DK, int OPT>
hipError_t launch_dk(const WyvParams& p, const GdnArgs& a, long nb, int nthr, hipStream_t s) {
    using T = typename Op<OPT>::T;
    const WyvLds<DK> L{p.max_depth};
    const size_t lds = (size_t)L.total() * sizeof(float);
    hipLaunchKernelGGL((wyv_kernel<DK, OPT>), dim3((unsigned)nb), dim3(nthr), lds, s, p, p.blob, static_cast<const T*>(a.q),
                       static_cast<const T*>(a.k), static_cast<const T*>(a.v), a.g, a.beta, a.state0,
                       static_cast<T*>(a.o));
    return hipGetLastError();
}

template <int OPT>
hipError_t launch_opt(int dk, const WyvParams& p, const GdnArgs& a, long nb, int nthr, hipStream_t s) {
    switch (dk) {
        case 16: return launch_dk<16, OPT>(p, a, nb, nthr, s);
        case 32: return launch_dk<32, OPT>(p, a, nb, nthr, s);
        case 64: return launch_dk<64, OPT>(p, a, nb, nthr, s);
        default: return launch_dk<128, OPT>(p, a, nb, nthr, s);
    }
}

}  // namespace

size_t wyv_lds_bytes(int d_k, int max_depth) {
    const int dm = max_depth < 1 ? 1 : max_depth;
    switch (d_k) {
        case 16: return (size_t)WyvLds<16>{dm}.total() * sizeof(float);
        case 32: return (size_t)WyvLds<32>{dm}.total() * sizeof(float);
        case 64: return (size_t)WyvLds<64>{dm}.total() * sizeof(float);
        default: return (size_t)WyvLds<128>{dm}.total() * sizeof(float);
    }
}

hipError_t launch_wyv(const lumo_gdn_dims& d, const lumo_tree_desc& desc, const GdnArgs& a, hipStream_t s) {
    const lumo_plan& pl = desc.plan;
    if (pl.total_nodes == 0) return hipSuccess;
    if (pl.max_depth > kWyvMaxDepth) return hipErrorNotSupported;
    WyvParams p;
    p.blob = desc.blob;
    p.o_node_off = pl.o_node_off;
    p.o_pre_row = pl.o_pre_row;
    p.o_pre_depth = pl.o_pre_depth;
    p.n_layers = d.n_layers;
    p.total_rows = pl.total_rows;
    p.h_k = d.h_k;
    p.h_v = d.h_v;
    p.d_v = d.d_v;
    p.group = d.h_v / d.h_k;
    p.n_vt = (d.d_v + 63) / 64;
    p.nwk = p.group * p.n_vt;
    p.n_wb = (p.nwk + kWpb - 1) / kWpb;
    p.max_depth = pl.max_depth < 1 ? 1 : pl.max_depth;
    p.qkn = (a.prep.flags & LUMO_PREP_QK_NORM) != 0;
    p.raw_gates = (a.prep.flags & LUMO_PREP_RAW_GATES) != 0;
    p.qk_eps = a.prep.qk_eps;
    p.a_log = a.prep.a_log;
    p.dt_bias = a.prep.dt_bias;
    const int nthr = 64 * (p.nwk < kWpb ? p.nwk : kWpb);
    const long nb = (long)d.n_req * d.n_layers * d.h_k * p.n_wb;
    return d.op_dtype == LUMO_BF16 ? launch_opt<1>(d.d_k, p, a, nb, nthr, s) : launch_opt<0>(d.d_k, p, a, nb, nthr, s);
}

}  // namespace lumo
