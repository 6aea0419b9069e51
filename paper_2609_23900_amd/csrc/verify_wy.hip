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
// One kernel. A block serves (request, layer, key head, NVH value heads of that key
// head's group) with two wavefronts per value head (64 value columns each; on small
// grids four of 32 columns), and walks the request's nodes in depth-first preorder, 32
// positions (a chunk) at a time:
//   staging   one chunk ahead with direct global-to-LDS loads: the chunk's key and
//             query rows plus the key rows of its path stack (the ancestry of its
//             first node), shared by the block; each wave's value rows.
//   Gram      MFMA between the candidates (path stack + chunk keys) and the chunk's
//             keys and queries. It does not depend on the value head: one 32 x 32
//             output tile per wave, into LDS.
//   R0 [K|Q]  MFMA against the wave's R0 columns, loaded once per block as B
//             fragments; a permlane32 swap leaves one value column per lane.
//   records   per node of the wave's head: the decay products along the ancestry and
//             {row, depth, beta, gamma, k.q, A[0..D), B[0..D)} with
//             A_m = beta Gamma(a_m->t) k_{a_m}.k_t, B_m = Gamma(a_m->t) k_{a_m}.q_t.
//   recursion the chunk in preorder with the deltas of the current path in registers
//             (the preorder path stack is exactly the ancestry).
// This replaces sequential scans; the arithmetic differs from them in rounding only
// (tolerance-level, not bitwise). The commit stays a sequential replay.
//
// Fused conv (CONV): the key, query and value rows are the tree conv's outputs of x
// rows, never stored. The block stages raw x rows where it would stage the rows, and at
// each chunk its threads (two channels each) walk the chunk's nodes in preorder with the
// raw x of the current root path kept by depth in LDS, so every node's window (its three
// nearest ancestors, or history entries) is at hand; the conv outputs replace the raw
// rows in place, and the keys of the root path are kept by depth for the next chunk's
// path-stack rows. The pending path's keys and values are convolved along the path, and
// the block publishes its slice of the history (one block per key head, so no other
// block reads that slice).
//
// Deferred publication (PEND): before the slab is split, each wave replays the previous
// iteration's accepted path on it with the sequential update (Eq. (2)-(3), one path
// node at a time, in fp32), stores it back to the state bank, and verifies from it. The
// state is then read once and written once per iteration; the publication of Alg. 1
// still precedes the verification that depends on it, per state tile.
#include "device_common.h"
#include "internal.h"
#include "launch.h"
#include "verify_wy.h"

namespace lumo {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;

constexpr int kD = 128;                // d_k = d_v
constexpr int kTile = kPreChunk;       // nodes per chunk = MFMA tile rows
constexpr int kStack = kPreStack;      // path-stack candidate slots (depth index < 16)
constexpr int kCand = kStack + kTile;  // Gram rows: stack slots, then the chunk's nodes
constexpr int kGS = 2 * kTile + 1;     // Gram row stride in floats: [chunk keys | chunk queries], padded
static_assert(kTile == 32, "one MFMA tile of nodes per chunk");

template <int D> struct Rec {
    static constexpr int kWords = 8 + 2 * D;  // {row, depth, beta, gamma, k.q, 0, 0, 0, A[D], B[D]}
};

struct WyParams {
    const int32_t* blob;
    int32_t o_node_off, o_pre_row, o_pre_depth, o_pre_ci, o_chunk_off, o_chunk_stack;
    int32_t n_layers, total_rows, h_k, h_v, group;
    int32_t raw_gates;  // g and beta hold raw inputs (operand preparation)
    float qk_eps;       // query/key normalisation constant (QKN kernels)
    const float* a_log;
    const float* dt_bias;
};

// The previous iteration's accepted path, published into the state bank before the
// verification reads it (deferred publication).
struct PendParams {
    const int32_t* blob;  // the previous iteration's plan
    int32_t o_node_off, o_row, total_rows, max_path;
    const int32_t* path_out;
    const int32_t* path_len;
    const uint16_t* k;
    const uint16_t* v;
    const float* g;
    const float* beta;
    float* state;
};
constexpr int kPend = 16;  // path entries staged per round of the deferred publication

// Fused conv (CONV kernels): x rows hold the channels q | k | v (value head h at
// 2 h_k d + h d); w [layers][channels][4], tap 3 the newest; bias nullable.
struct ConvFuseParams {
    const uint16_t* x;
    uint16_t* hist;          // [req][layers][3][channels], published in place
    const uint16_t* x_prev;  // the pending path's rows
    const float* w;
    const float* bias;
    int32_t channels, act;
};

// Block-shared staging of one chunk: [key 32 | query 32 | path-stack key 16] rows of
// 16 slots of 8 bf16; key block kb of row n sits in slot kb ^ (n & 15), so the
// fragment reads of a half-wave (32 rows, one key block) spread over all banks.
constexpr int kTileRows = 2 * kTile + kStack;
struct KQTile {
    uint4 slot[kTileRows * 16];
};

// Per-lane view of one chunk. Lanes 0..31 and 32..63 both describe node t = lane % 32
// (depth, candidate slots, beta); g is that of the lane's row (see lane_info).
template <int D>
struct LaneInfo {
    int dep;
    uint32_t ci[D / 4];
    float g, b;
};

template <int R> struct RoleTag {
    static constexpr int value = R;
};

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 w) { return __builtin_bit_cast(bf16x8, w); }


// Two waves per SIMD for D = 8 (79 KB of LDS per 4-wave block). With D = 16 (and no
// fused conv) the two waves of a value head share one record buffer (the even wave
// writes it, a barrier publishes it), which keeps the 4-wave block at 76 KB, so two
// blocks fit a CU, and the block is compiled for two waves per SIMD (256 registers).
// The fused conv's D = 16 instance keeps per-wave buffers and one wave per SIMD.
// PEND: the state bank (state0 = pd.state) first receives the replay of the previous
// iteration's accepted path (Eq. (2)-(3) per path node), is stored back, and the
// verification then starts from it; requests without nodes are published only.
// QKN: every query and key row x is used as x / sqrt(|x|^2 + eps) (Sec. IV-B). The
// bf16 rows stay as they are in LDS and the MFMA products; the per-row factors scale
// the Gram entries, R0 k, R0 q and k.q in the records, and the pending path's keys.
// CW = 32 (small grids): four waves per value head, 32 state columns each, so that a
// call with fewer blocks than CUs still has a wave on every SIMD and each wave's walk
// (state slab, publication, products) is half as long. A wave's lanes l and l + 32
// then hold the same column: l < 32 forms the ancestor sum of A and the delta, l >= 32
// the sum of B and the output. Every value is computed with the operations, and in the
// order, of the 64-column form, so both give the same bits.
template <int D, int NVH, bool PEND, bool QKN, bool CONV, int CW = 64>
__global__ __launch_bounds__(64 * (CW == 64 ? 2 : 4) * NVH, (D == 8 || CW == 32 || (!CONV && NVH == 2)) ? 2 : 1) void wy_kernel(WyParams p, const uint16_t* __restrict__ kmat,
                                                    const uint16_t* __restrict__ qmat,
                                                    const uint16_t* __restrict__ vmat, const float* __restrict__ gmat,
                                                    const float* __restrict__ bmat, const float* __restrict__ state0,
                                                    uint16_t* __restrict__ out, PendParams pd, ConvFuseParams cf) {
    const int wy_bid = (int)blockIdx.x, wy_nblk = (int)gridDim.x;
#include "verify_wy_body.inc"
}

// Two calls of the 32-column form with deferred publication in one launch: blocks
// [0, na) serve call a, the others call b, each block exactly as a wy_kernel block of
// its own call (its plan, operands, state bank and pending path). Calls that share no
// output then run side by side: a layer's verification next to the publication of the
// pending path into another layer's state bank, which has no tree to verify.
struct WyCall {
    WyParams p;
    const uint16_t* k;
    const uint16_t* q;
    const uint16_t* v;
    const float* g;
    const float* beta;
    uint16_t* out;
    PendParams pd;
};

template <int DD, bool QQ>
__global__ __launch_bounds__(256, 2) void wy_pair_kernel(WyCall ca, WyCall cb, int na) {
    constexpr int D = DD, NVH = 1, CW = 32;
    constexpr bool PEND = true, QKN = QQ, CONV = false;
    const bool first = (int)blockIdx.x < na;  // uniform
    const WyCall& c = first ? ca : cb;
    const WyParams p = c.p;
    const uint16_t* __restrict__ kmat = c.k;
    const uint16_t* __restrict__ qmat = c.q;
    const uint16_t* __restrict__ vmat = c.v;
    const float* __restrict__ gmat = c.g;
    const float* __restrict__ bmat = c.beta;
    const PendParams pd = c.pd;
    const float* __restrict__ state0 = pd.state;
    uint16_t* __restrict__ out = c.out;
    const ConvFuseParams cf{};
    const int wy_bid = first ? (int)blockIdx.x : (int)blockIdx.x - na;
    const int wy_nblk = first ? na : (int)gridDim.x - na;
#include "verify_wy_body.inc"
}

template <int D, int NVH, bool PEND, bool QKN, bool CONV = false, int CW = 64>
hipError_t launch_wy_kernel(const lumo_gdn_dims& d, const WyParams& p, const GdnArgs& a, hipStream_t s,
                            const PendParams& pp, const ConvFuseParams& cf = ConvFuseParams{}) {
    const long nb = (long)d.n_req * d.n_layers * d.h_k * (p.group / NVH);
    hipLaunchKernelGGL((wy_kernel<D, NVH, PEND, QKN, CONV, CW>), dim3((unsigned)nb), dim3(64 * (128 / CW) * NVH), 0, s, p,
                       static_cast<const uint16_t*>(a.k), static_cast<const uint16_t*>(a.q),
                       static_cast<const uint16_t*>(a.v), a.g, a.beta, PEND ? pp.state : a.state0,
                       static_cast<uint16_t*>(a.o), pp, cf);
    return hipGetLastError();
}

WyParams wy_params(const lumo_gdn_dims& d, const lumo_tree_desc& desc, const GdnArgs& a) {
    const lumo_plan& pl = desc.plan;
    WyParams p;
    p.blob = desc.blob;
    p.o_node_off = pl.o_node_off;
    p.o_pre_row = pl.o_pre_row;
    p.o_pre_depth = pl.o_pre_depth;
    p.o_pre_ci = pl.o_pre_ci;
    p.o_chunk_off = pl.o_chunk_off;
    p.o_chunk_stack = pl.o_chunk_stack;
    p.n_layers = d.n_layers;
    p.total_rows = pl.total_rows;
    p.h_k = d.h_k;
    p.h_v = d.h_v;
    p.group = d.h_v / d.h_k;
    p.raw_gates = (a.prep.flags & LUMO_PREP_RAW_GATES) != 0;
    p.qk_eps = a.prep.qk_eps;
    p.a_log = a.prep.a_log;
    p.dt_bias = a.prep.dt_bias;
    return p;
}

template <int D, bool PEND>
hipError_t launch_wy_d(const lumo_gdn_dims& d, const lumo_tree_desc& desc, const GdnArgs& a, hipStream_t s,
                       const PendParams& pp) {
    const WyParams p = wy_params(d, desc, a);
    // one block per (request, layer, key head, pair of value heads): the pair's waves
    // share the staged key and query rows and the Gram. Grids of fewer pair blocks than
    // CUs (one layer of a batch, few requests) take one value head per block instead,
    // with four waves of 32 columns: four times the waves, each with half the work on
    // its critical path, at the cost of a Gram per head.
    const bool qkn = (a.prep.flags & LUMO_PREP_QK_NORM) != 0;
    const long pair_blocks = (long)d.n_req * d.n_layers * d.h_k * (p.group / 2);
    if (p.group % 2 == 0 && pair_blocks >= 256)
        return qkn ? launch_wy_kernel<D, 2, PEND, true>(d, p, a, s, pp) : launch_wy_kernel<D, 2, PEND, false>(d, p, a, s, pp);
    return qkn ? launch_wy_kernel<D, 1, PEND, true, false, 32>(d, p, a, s, pp)
               : launch_wy_kernel<D, 1, PEND, false, false, 32>(d, p, a, s, pp);
}

}  // namespace

PendParams pend_params(const PendArgs& pend) {
    const lumo_plan& pl = pend.desc->plan;
    PendParams pp;
    pp.blob = pend.desc->blob;
    pp.o_node_off = pl.o_node_off;
    pp.o_row = pl.o_row;
    pp.total_rows = pl.total_rows;
    pp.max_path = pend.max_path;
    pp.path_out = pend.path_out;
    pp.path_len = pend.path_len;
    pp.k = static_cast<const uint16_t*>(pend.k);
    pp.v = static_cast<const uint16_t*>(pend.v);
    pp.g = pend.g;
    pp.beta = pend.beta;
    pp.state = pend.state;
    return pp;
}

hipError_t launch_wy(const lumo_gdn_dims& d, const lumo_tree_desc& desc, const GdnArgs& a, hipStream_t s,
                     const PendArgs* pend) {
    if (desc.plan.max_depth > kStack + 1) return hipErrorNotSupported;
    // path-stack registers: depths 0..7 suffice when no path is longer than 9 nodes
    const bool d8 = desc.plan.max_depth <= 9;
    if (!pend) {
        if (desc.plan.total_nodes == 0) return hipSuccess;
        const PendParams none{};
        return d8 ? launch_wy_d<8, false>(d, desc, a, s, none) : launch_wy_d<16, false>(d, desc, a, s, none);
    }
    if (d.n_req == 0) return hipSuccess;  // requests without nodes are still published
    const PendParams pp = pend_params(*pend);
    return d8 ? launch_wy_d<8, true>(d, desc, a, s, pp) : launch_wy_d<16, true>(d, desc, a, s, pp);
}

hipError_t launch_wy_conv(const lumo_gdn_dims& d, const lumo_tree_desc& desc, const GdnArgs& a, hipStream_t s,
                          const PendArgs& pend, const ConvFuseArgs& c) {
    if (desc.plan.max_depth > kStack + 1 || d.h_v != 2 * d.h_k) return hipErrorNotSupported;
    if (d.n_req == 0) return hipSuccess;
    const bool d8 = desc.plan.max_depth <= 9;
    const WyParams p = wy_params(d, desc, a);
    const PendParams pp = pend_params(pend);
    ConvFuseParams cf;
    cf.x = static_cast<const uint16_t*>(c.x);
    cf.hist = static_cast<uint16_t*>(c.hist);
    cf.x_prev = static_cast<const uint16_t*>(c.x_prev);
    cf.w = c.w;
    cf.bias = c.bias;
    cf.channels = c.channels;
    cf.act = c.act;
    const bool qkn = (a.prep.flags & LUMO_PREP_QK_NORM) != 0;
    if (d8)
        return qkn ? launch_wy_kernel<8, 2, true, true, true>(d, p, a, s, pp, cf)
                   : launch_wy_kernel<8, 2, true, false, true>(d, p, a, s, pp, cf);
    return qkn ? launch_wy_kernel<16, 2, true, true, true>(d, p, a, s, pp, cf)
               : launch_wy_kernel<16, 2, true, false, true>(d, p, a, s, pp, cf);
}

hipError_t launch_wy_pair(const lumo_gdn_dims& da, const lumo_tree_desc& desca, const GdnArgs& aa, const PendArgs& pa,
                          const lumo_gdn_dims& db, const lumo_tree_desc& descb, const GdnArgs& ab, const PendArgs& pb,
                          hipStream_t s) {
    if (desca.plan.max_depth > kStack + 1 || descb.plan.max_depth > kStack + 1) return hipErrorNotSupported;
    const bool qkn = (aa.prep.flags & LUMO_PREP_QK_NORM) != 0;
    if (qkn != ((ab.prep.flags & LUMO_PREP_QK_NORM) != 0)) return hipErrorNotSupported;
    const bool d8 = desca.plan.max_depth <= 9 && descb.plan.max_depth <= 9;
    WyCall ca{wy_params(da, desca, aa), static_cast<const uint16_t*>(aa.k), static_cast<const uint16_t*>(aa.q),
              static_cast<const uint16_t*>(aa.v), aa.g, aa.beta, static_cast<uint16_t*>(aa.o), pend_params(pa)};
    WyCall cb{wy_params(db, descb, ab), static_cast<const uint16_t*>(ab.k), static_cast<const uint16_t*>(ab.q),
              static_cast<const uint16_t*>(ab.v), ab.g, ab.beta, static_cast<uint16_t*>(ab.o), pend_params(pb)};
    const long na = (long)da.n_req * da.n_layers * da.h_v;  // one value head per block
    const long nb = (long)db.n_req * db.n_layers * db.h_v;
    if (na + nb == 0) return hipSuccess;
    const dim3 grid((unsigned)(na + nb));
    if (d8) {
        if (qkn)
            hipLaunchKernelGGL((wy_pair_kernel<8, true>), grid, dim3(256), 0, s, ca, cb, (int)na);
        else
            hipLaunchKernelGGL((wy_pair_kernel<8, false>), grid, dim3(256), 0, s, ca, cb, (int)na);
    } else {
        if (qkn)
            hipLaunchKernelGGL((wy_pair_kernel<16, true>), grid, dim3(256), 0, s, ca, cb, (int)na);
        else
            hipLaunchKernelGGL((wy_pair_kernel<16, false>), grid, dim3(256), 0, s, ca, cb, (int)na);
    }
    return hipGetLastError();
}

}  // namespace lumo
