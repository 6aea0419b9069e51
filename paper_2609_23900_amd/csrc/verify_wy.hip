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
    static_assert(!CONV || (NVH == 2 && PEND && CW == 64), "the fused conv serves two value heads per block, with publication");
    static_assert(CW == 64 || (CW == 32 && NVH == 1), "32-column waves serve one value head per block");
    constexpr int W = Rec<D>::kWords;
    constexpr int WPH = kD / CW;       // waves per value head
    constexpr int NCT = CW / 16;       // 16-column MFMA tiles per wave
    constexpr int SPN = CW / 8;        // 16-byte value slots per node and wave
    constexpr bool AB = CW == 32;      // lane halves split the recursion's sums
    constexpr int NW = WPH * NVH;      // waves per block
    constexpr int nthr = 64 * NW;
    // the waves of a value head share its records (D = 16 without the fused conv, and
    // the four waves of 32 columns)
    constexpr bool SHR = (D == 16 && !CONV) || AB;
    // LDS, one object per role: the compiler orders LDS reads after the direct
    // global-to-LDS copies only where they may touch the same object.
    __shared__ KQTile tile;                        // block: chunk keys, queries, path-stack keys
    __shared__ __attribute__((aligned(16))) float G[kCand * kGS];  // block: Gram [candidate][chunk key | chunk query]
    // per wave (SHR: per value head): the chunk's coefficient records
    __shared__ __attribute__((aligned(16))) float recs[SHR ? NVH : NW][kTile * W];
    __shared__ float alphas[NW][64];               // per wave: exp(g) of the candidates
    // per wave: value rows, then outputs; double-buffered (CONV: single, for the caches)
    __shared__ uint4 vbufs[NW][CONV ? 1 : 2][kTile * SPN];
    // CONV: raw x of the current root path by depth (rows 0..2 the history, row 3 + d
    // depth d), two channels per thread; conv outputs of the root path's keys by depth
    __shared__ uint32_t rawc[CONV ? D + 4 : 1][CONV ? nthr : 1];
    __shared__ uint32_t kcache[CONV ? D + 1 : 1][CONV ? 64 : 1];
    __shared__ float nrm[kTileRows];               // QKN: 1/|row| of [stack keys 16 | chunk keys 32 | queries 32]
    const int tid = (int)threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: head and half in SGPRs
    const int lane = tid & 63;
    float* wrec = recs[SHR ? wave / WPH : wave];
    float* walpha = alphas[wave];
    const bool rec_writer = !SHR || wave % WPH == 0;  // uniform

    // The blocks of one (request, layer) share its gate rows (g and beta of every head
    // of a row sit in one line) and, with several blocks per key head, the key and
    // query rows: they run on one XCD, whose L2 serves them to all. Consecutive
    // (request, layer) units go to different XCDs, so requests of very different sizes
    // (a run of chains, then a run of trees) spread over the whole device.
    const int pairs = p.group / NVH;
    int blk = xcd_units((int)blockIdx.x, (int)gridDim.x, p.h_k * pairs);
    const int pp = blk % pairs;
    blk /= pairs;
    const int hk = blk % p.h_k;
    blk /= p.h_k;
    const int l = blk % p.n_layers;
    const int r = blk / p.n_layers;
    const int h = hk * p.group + pp * NVH + wave / WPH;
    const int j0 = CW * (wave % WPH);
    const bool rawg = p.raw_gates != 0;  // uniform
    const float alog = rawg ? p.a_log[l * p.h_v + h] : 0.f;
    const float dtb = rawg ? p.dt_bias[l * p.h_v + h] : 0.f;
    const int base = p.blob[p.o_node_off + r];
    const int N = p.blob[p.o_node_off + r + 1] - base;
    int plen = 0;  // pending path length; an empty or invalid path leaves the state as it is
    int pp0 = 0;   // node of pending path entry min(lane % kPend, max_path - 1), loaded with the length
    if constexpr (PEND) {
        plen = pd.path_len[r];
        pp0 = pd.path_out[(long)r * pd.max_path + min(lane % kPend, pd.max_path - 1)];
        if (plen > pd.max_path || pd.blob[pd.o_node_off + r + 1] <= pd.blob[pd.o_node_off + r]) plen = 0;
    }
    if (N <= 0 && plen <= 0) return;  // uniform over the block
    const int32_t* prow = p.blob + p.o_pre_row + base;
    const int32_t* pdep = p.blob + p.o_pre_depth + base;
    const uint32_t* pci = reinterpret_cast<const uint32_t*>(p.blob + p.o_pre_ci) + (long)kPreCiWords * base;
    const int32_t* stacks = p.blob + p.o_chunk_stack + (long)kStack * p.blob[p.o_chunk_off + r];
    const long krow0 = (long)l * p.total_rows;
    const int t = lane % kTile;  // node of this lane in the chunk views
    // Inside the chunk loop the lane index is re-laundered at every chunk, so values
    // derived from it (LDS addresses and offsets) are recomputed rather than kept live
    // across the loop, which would not fit in the registers.
    int ln = lane;
    int tn = t;
    // CONV: x row stride and the block's channel groups (queries, keys, values)
    const long xc = CONV ? cf.channels : 0;
    const int qoff = hk * kD, koff = (p.h_k + hk) * kD, voff = 2 * p.h_k * kD;

    // Rows of the chunk at c0 as seen by this lane: n = node t's (every lane; positions
    // past the end repeat the last node, so padding slots are exact copies of it) and
    // s = path-stack slot lane%16's, -1 beyond the first node's depth (clamped to row 0
    // where used: those Gram rows are never referenced). Both loads are unconditional
    // and nothing is computed from them until they are used.
    struct Rows {
        int n, s;
    };
    auto lane_rows = [&](int c0) {
        Rows rw;
        rw.n = prow[min(c0 + t, N - 1)];
        rw.s = stacks[(c0 / kTile) * kStack + (lane & (kStack - 1))];
        return rw;
    };
    // g of lane rows (stack slot lane-32's on lanes 32..47, node t's otherwise), node t's
    // depth, candidate slots and beta
    auto lane_info = [&](int c0, const Rows& rw, LaneInfo<D>& li) {
        const int pos = min(c0 + t, N - 1);
        li.dep = pdep[pos];
#pragma unroll
        for (int w = 0; w < D / 4; ++w) li.ci[w] = pci[(long)kPreCiWords * pos + w];
        const int grow = (lane >= kTile && lane < kTile + kStack) ? max(rw.s, 0) : rw.n;
        li.g = gmat[(krow0 + grow) * p.h_v + h];
        li.b = bmat[(krow0 + rw.n) * p.h_v + h];
    };
    // Block-shared tile rows of the chunk. In round j a wave fills tile rows nr0 .. nr0+3
    // (16 slots each), so the four source rows are read with readlane: no LDS access,
    // hence no ordering behind copies still in flight.
    constexpr int kTileRounds = kTileRows * 16 / nthr;
    auto tile_issue = [&](const Rows& rw) {
        int ln = lane;
        asm volatile("" : "+v"(ln));  // recomputed per call rather than kept live across the loop
#pragma unroll
        for (int j = 0; j < kTileRounds; ++j) {
            const int nr0 = (j * nthr + 64 * wave) >> 4;  // uniform
            // a round lies wholly in the key/query rows or wholly in the stack rows
            constexpr int kRoundRows = nthr / 16;
            static_assert(2 * kTile % kRoundRows == 0, "rounds do not straddle the stack rows");
            const bool stack_round = j * kRoundRows >= 2 * kTile;  // compile-time per round
            int rq[4];
#pragma unroll
            for (int k4 = 0; k4 < 4; ++k4) {
                const int nr = nr0 + k4;
                rq[k4] = stack_round ? max(__builtin_amdgcn_readlane(rw.s, nr - 2 * kTile), 0)
                                     : __builtin_amdgcn_readlane(rw.n, nr % kTile);
            }
            const int g4 = ln >> 4;
            const int src = g4 == 0 ? rq[0] : g4 == 1 ? rq[1] : g4 == 2 ? rq[2] : rq[3];
            const int nr = nr0 + g4;
            const int kb = (ln & 15) ^ (nr & 15);
            if constexpr (CONV) {
                // raw x rows; the path-stack rows come from the key cache instead
                if (stack_round) continue;
                __builtin_amdgcn_global_load_lds(cf.x + (krow0 + src) * xc + (nr >= kTile ? qoff : koff) + 8 * kb,
                                                 (lds_void*)&tile.slot[j * nthr + 64 * wave], 16, 0, 0);
                continue;
            }
            const uint16_t* mat = (!stack_round && nr >= kTile) ? qmat : kmat;
            __builtin_amdgcn_global_load_lds(mat + ((krow0 + src) * p.h_k + hk) * kD + 8 * kb,
                                             (lds_void*)&tile.slot[j * nthr + 64 * wave], 16, 0, 0);
        }
    };
    // Block barrier after this wave's LDS writes have completed. Unlike __syncthreads it
    // does not wait for global memory operations (copies into other LDS objects, output
    // stores) that nothing across the barrier depends on.
    auto lds_barrier = [&]() {
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
    };
    // The recursion leaves node n's output (bf16, this wave's CW columns) in place of its
    // value entries; a chunk's output rows then go out as 16-byte stores (slot q: node
    // q / SPN, columns j0 + 8 (q % SPN) ..), rows taken from the records. Padding slots
    // repeat the last node's row and values. nodes = 16 when the second half was not
    // computed.
    constexpr int kVRounds = kTile * SPN / 64;
    auto flush = [&](const uint4* ob, int nodes) {
#pragma unroll
        for (int i = 0; i < kVRounds; ++i) {
            if (64 * i >= nodes * SPN) break;  // uniform
            const int q = 64 * i + ln;
            const uint4 val = ob[q];
            const int rn = __float_as_int(wrec[(q / SPN) * W]);
            *reinterpret_cast<uint4*>(out + ((krow0 + rn) * p.h_v + h) * kD + j0 + 8 * (q % SPN)) = val;
        }
    };
    // the wave's value rows: slot q = 64 i + lane holds node q / SPN, columns
    // j0 + 8 (q % SPN) .. + 7
    auto v_issue = [&](const Rows& rw, uint4* dst) {
        int ln = lane;
        asm volatile("" : "+v"(ln));  // recomputed per call rather than kept live across the loop
        int rn[kVRounds];
#pragma unroll
        for (int i = 0; i < kVRounds; ++i) rn[i] = __shfl(rw.n, (64 * i + ln) / SPN);
#pragma unroll
        for (int i = 0; i < kVRounds; ++i) {
            const int q = 64 * i + ln;
            const uint16_t* src = CONV ? cf.x + (krow0 + rn[i]) * xc + voff + h * kD + j0 + 8 * (q % SPN)
                                       : vmat + ((krow0 + rn[i]) * p.h_v + h) * kD + j0 + 8 * (q % SPN);
            __builtin_amdgcn_global_load_lds(src, (lds_void*)&dst[64 * i], 16, 0, 0);
        }
    };

    // CONV walks: thread tid serves x channels 2 (tid % 4), +1 of 8-channel slot
    // cs = tid / 4: keys (cs < 16), queries (cs < 32), values of wave (cs - 32) / 8.
    struct Taps {
        float lo[4], hi[4], blo, bhi;
    };
    auto walk_channel = [&]() -> int {
        const int cs = tid >> 2, pt = tid & 3;
        if (cs < 16) return koff + 8 * cs + 2 * pt;
        if (cs < 32) return qoff + 8 * (cs - 16) + 2 * pt;
        const int vw = (cs - 32) >> 3;
        const int hv = hk * p.group + pp * NVH + (vw >> 1);
        return voff + hv * kD + 64 * (vw & 1) + 8 * ((cs - 32) & 7) + 2 * pt;
    };
    auto load_taps = [&](Taps& tp) {
        const long c = (long)l * xc + walk_channel();
        const float4 a = *reinterpret_cast<const float4*>(cf.w + c * 4);
        const float4 b = *reinterpret_cast<const float4*>(cf.w + (c + 1) * 4);
        tp.lo[0] = a.x; tp.lo[1] = a.y; tp.lo[2] = a.z; tp.lo[3] = a.w;
        tp.hi[0] = b.x; tp.hi[1] = b.y; tp.hi[2] = b.z; tp.hi[3] = b.w;
        tp.blo = cf.bias ? cf.bias[c] : 0.f;
        tp.bhi = cf.bias ? cf.bias[c + 1] : 0.f;
    };
    // act(bias + sum_t w_t window_t) of a channel pair, taps oldest first and the node's
    // own entry last, fp32, then one cast: the conv kernels' arithmetic
    auto conv2 = [&](const Taps& tp, uint32_t w0, uint32_t w1, uint32_t w2, uint32_t xr) -> uint32_t {
        float lo = tp.blo, hi = tp.bhi;
        lo = __builtin_fmaf(tp.lo[0], bf16_lo(w0), lo);
        hi = __builtin_fmaf(tp.hi[0], bf16_hi(w0), hi);
        lo = __builtin_fmaf(tp.lo[1], bf16_lo(w1), lo);
        hi = __builtin_fmaf(tp.hi[1], bf16_hi(w1), hi);
        lo = __builtin_fmaf(tp.lo[2], bf16_lo(w2), lo);
        hi = __builtin_fmaf(tp.hi[2], bf16_hi(w2), hi);
        lo = __builtin_fmaf(tp.lo[3], bf16_lo(xr), lo);
        hi = __builtin_fmaf(tp.hi[3], bf16_hi(xr), hi);
        if (cf.act == 1) {  // SiLU, as in the conv kernels
            lo = lo * __builtin_amdgcn_rcpf(1.f + __expf(-lo));
            hi = hi * __builtin_amdgcn_rcpf(1.f + __expf(-hi));
        }
        return f32x2_to_bf16x2(lo, hi);
    };
    // the chunk's nodes in preorder: window from the root-path cache, the raw entry into
    // the cache at the node's depth, the conv output over the raw entry (tile rows,
    // value buffers), the key into the key cache. Padding slots repeat the last node and
    // redo it exactly.
    // A wave's channels are all keys (wave 0), all queries (wave 1) or all values, so the
    // walk is specialised per role. Node n + 1's window and raw entry are read before
    // node n's writes: in preorder the next depth is at most d + 1, so the only entry
    // node n writes that node n + 1 can need is its own raw entry (the newest window
    // entry of a child), taken from the register.
    static_assert(!CONV || nthr == 256, "one role per wave: keys, queries, two waves of values");
    auto conv_walk_role = [&](const Taps& tp, const LaneInfo<D>& li, auto role) {
        constexpr int R = decltype(role)::value;
        const int cs = tid >> 2, pt = tid & 3;
        auto px = [&](int n) -> uint32_t* {
            if constexpr (R == 0) return reinterpret_cast<uint32_t*>(&tile.slot[n * 16 + (cs ^ (n & 15))]) + pt;
            else if constexpr (R == 1)
                return reinterpret_cast<uint32_t*>(&tile.slot[(kTile + n) * 16 + ((cs - 16) ^ (n & 15))]) + pt;
            else return reinterpret_cast<uint32_t*>(&vbufs[(cs - 32) >> 3][0][8 * n + ((cs - 32) & 7)]) + pt;
        };
        int d = __builtin_amdgcn_readlane(li.dep, 0);
        uint32_t w0 = rawc[d][tid], w1 = rawc[d + 1][tid], w2 = rawc[d + 2][tid], xr = *px(0);
#pragma unroll 4
        for (int n = 0; n < kTile; ++n) {
            const int nn = n + 1 < kTile ? n + 1 : n;
            const int dn = __builtin_amdgcn_readlane(li.dep, nn);
            const uint32_t v0 = rawc[dn][tid], v1 = rawc[dn + 1][tid], v2 = rawc[dn + 2][tid];
            const uint32_t xn = *px(nn);
            const uint32_t y = conv2(tp, w0, w1, w2, xr);
            rawc[d + 3][tid] = xr;
            *px(n) = y;
            if constexpr (R == 0) kcache[d][tid] = y;
            w0 = v0;
            w1 = v1;
            w2 = dn == d + 1 ? xr : v2;
            xr = xn;
            d = dn;
        }
    };
    auto conv_walk = [&](const Taps& tp, const LaneInfo<D>& li) {
        const int role = __builtin_amdgcn_readfirstlane(tid >> 6);
        if (role == 0) conv_walk_role(tp, li, RoleTag<0>{});
        else if (role == 1) conv_walk_role(tp, li, RoleTag<1>{});
        else conv_walk_role(tp, li, RoleTag<2>{});
    };
    // the root-path caches at the start of the walk: the history, and keys and
    // path-stack rows cleared (finite; rows past a node's depth are masked, not skipped)
    auto conv_cache_init = [&](uint32_t a0, uint32_t a1, uint32_t a2) {
        rawc[0][tid] = a0;
        rawc[1][tid] = a1;
        rawc[2][tid] = a2;
        if (tid < 64) {
#pragma unroll
            for (int m = 0; m <= D; ++m) kcache[m][tid] = 0u;
        }
        static_assert(kStack * 16 == nthr || !CONV, "one 16-byte piece of the stack rows per thread");
        tile.slot[2 * kTile * 16 + tid] = make_uint4(0, 0, 0, 0);
    };
    // the next chunk's path-stack rows: the keys of the root path by depth
    auto stack_from_cache = [&]() {
        if (tid < 64) {
            const int cs = tid >> 2, pt = tid & 3;
            constexpr int ns = D + 1 < kStack ? D + 1 : kStack;
#pragma unroll
            for (int m = 0; m < ns; ++m)
                reinterpret_cast<uint32_t*>(&tile.slot[(2 * kTile + m) * 16 + (cs ^ m)])[pt] = kcache[m][tid];
        }
    };

    // R0 as B fragments of the 16x16x32 MFMA: column n = lane%16 of tile ct is state
    // column j0 + NCT n + ct, and key block kb holds keys 32 kb + 8 (lane/16) + e. A lane
    // thus holds NCT adjacent columns of each of its keys: one 16-byte (CW = 32: 8-byte)
    // load and store per key. After the lane exchange of the products, lane l serves
    // state column j0 + pc, pc = NCT (l % 16) + (l / 16) % NCT.
    const float* S = state0 + (((long)r * p.n_layers + l) * p.h_v + h) * (long)(kD * kD);
    const float* Sl = S + (long)(8 * (lane / 16)) * kD + j0 + NCT * (lane % 16);
    uint32_t raw[NCT][kD / 32][8];
    auto slab_load = [&](int kb) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            if constexpr (NCT == 4) {
                const uint4 w = *reinterpret_cast<const uint4*>(Sl + (long)(32 * kb + e) * kD);
                raw[0][kb][e] = w.x;
                raw[1][kb][e] = w.y;
                raw[2][kb][e] = w.z;
                raw[3][kb][e] = w.w;
            } else {
                const uint2 w = *reinterpret_cast<const uint2*>(Sl + (long)(32 * kb + e) * kD);
                raw[0][kb][e] = w.x;
                raw[1][kb][e] = w.y;
            }
        }
    };
    // The chunk's rows are loaded first and half the state slab behind them, so that the
    // row-dependent copies below wait for the rows only (16 loads issued after them)
    // while the slab is already in flight; then the other half.
    // Deferred publication: the pending path's key rows (block-shared, in the Gram's
    // space) and the wave's value entries (in its record space; with 32 columns in its
    // second value buffer) are staged kPend entries at a time; lane e holds entry e's
    // decay and beta. Each entry applies
    //   u = R k,  delta = beta (v - alpha u),  R <- alpha R + delta k
    // to the slab in registers (lane: NCT columns x 32 keys; u summed over the four lane
    // rows that share a column), then the slab is stored back.
    auto pend_publish = [&]() {
        const int pbase = pd.blob[pd.o_node_off + r];
        const int pn = pd.blob[pd.o_node_off + r + 1] - pbase;
        const int32_t* ppath = pd.path_out + (long)r * pd.max_path;
        const long prow0 = (long)l * pd.total_rows;
        uint4* kst = reinterpret_cast<uint4*>(G);       // kPend key rows x 16 slots
        // kPend entries x CW values (SPN slots) in the record space; with shared records
        // each wave of the head takes its own half of it; 32-column waves use their second
        // value buffer (filled only by the first chunk's loop)
        static_assert(AB || !SHR || kTile * W >= 2 * (kPend * 64 / 2), "two staging areas fit one record buffer");
        static_assert(!AB || kTile * SPN >= kPend * SPN, "the staging fits a value buffer");
        float* vstage = AB ? reinterpret_cast<float*>(vbufs[wave][1])
                           : wrec + (SHR ? (wave & 1) * (kPend * 64 / 2) : 0);
        uint4* vst = reinterpret_cast<uint4*>(vstage);
        const uint16_t* vsh = reinterpret_cast<const uint16_t*>(vstage);
        // CONV: this thread's channels of the old history (the chain conv's first window,
        // rolled along the path) and of the published one, the last three of (old
        // history, the path's raw x rows)
        uint32_t hw0 = 0, hw1 = 0, hw2 = 0, hn0 = 0, hn1 = 0, hn2 = 0;
        uint16_t* hsl = nullptr;
        Taps tpp;
        if constexpr (CONV) {
            const int c = walk_channel();
            hsl = cf.hist + ((long)r * p.n_layers + l) * 3 * xc + c;
            hw0 = *reinterpret_cast<const uint32_t*>(hsl);
            hw1 = *reinterpret_cast<const uint32_t*>(hsl + xc);
            hw2 = *reinterpret_cast<const uint32_t*>(hsl + 2 * xc);
            int hrow = 0;  // lane j < 3: the row of path entry plen + j - 3, when there is one
            if (lane < 3 && plen + lane >= 3) {
                const int node = min(max(ppath[plen + lane - 3], 0), pn - 1);
                hrow = pd.blob[pd.o_row + pbase + node];
            }
            uint32_t hn[3];
#pragma unroll
            for (int j = 0; j < 3; ++j) {
                const int pos = plen + j;
                const int rowj = __builtin_amdgcn_readlane(hrow, j);
                hn[j] = pos >= 3 ? *reinterpret_cast<const uint32_t*>(cf.x_prev + (prow0 + rowj) * xc + c)
                                 : (pos == 1 ? hw1 : hw2);  // pos is at least 1
            }
            hn0 = hn[0];
            hn1 = hn[1];
            hn2 = hn[2];
            load_taps(tpp);
        }
        for (int e0 = 0; e0 < plen; e0 += kPend) {
            const int ne = min(plen - e0, kPend);
            if (e0 > 0) lds_barrier();  // every wave has read the previous entries' key rows
            // entry e0 + min(lane % kPend, ne - 1); the first round's nodes were loaded at the start
            const int pnode = e0 > 0 ? ppath[e0 + min(lane % kPend, ne - 1)]
                                     : (lane % kPend < ne ? pp0 : __builtin_amdgcn_readlane(pp0, ne - 1));
            const int node = min(max(pnode, 0), pn - 1);
            const int row = pd.blob[pd.o_row + pbase + node];
            const long gl = (prow0 + row) * p.h_v + h;
            float pgv = pd.g[gl], pb = pd.beta[gl];
            if (rawg) {
                pgv = raw_log_alpha(pgv, alog, dtb);
                pb = raw_beta(pb);
            }
            const float pa = __expf(pgv);
            constexpr int kPV = kPend * SPN / 64;  // value-staging rounds
            int rv[kPV];
#pragma unroll
            for (int i = 0; i < kPV; ++i) rv[i] = __shfl(row, (64 * i + lane) / SPN);
            constexpr int kKRounds = kPend * 16 / nthr;
#pragma unroll
            for (int j = 0; j < kKRounds; ++j) {
                const int nr0 = (j * nthr + 64 * wave) >> 4;  // uniform: this wave fills rows nr0 .. nr0+3
                int rq[4];
#pragma unroll
                for (int k4 = 0; k4 < 4; ++k4) rq[k4] = __builtin_amdgcn_readlane(row, nr0 + k4);
                const int g4 = lane >> 4;
                const int src = g4 == 0 ? rq[0] : g4 == 1 ? rq[1] : g4 == 2 ? rq[2] : rq[3];
                const uint16_t* ks = CONV ? cf.x_prev + (prow0 + src) * xc + koff + 8 * (lane & 15)
                                          : pd.k + ((prow0 + src) * p.h_k + hk) * kD + 8 * (lane & 15);
                __builtin_amdgcn_global_load_lds(ks, (lds_void*)&kst[j * nthr + 64 * wave], 16, 0, 0);
            }
#pragma unroll
            for (int i = 0; i < kPV; ++i) {
                const int q = 64 * i + lane;
                const uint16_t* vsrc = CONV ? cf.x_prev + (prow0 + rv[i]) * xc + voff + h * kD + j0 + 8 * (q % SPN)
                                            : pd.v + ((prow0 + rv[i]) * p.h_v + h) * kD + j0 + 8 * (q % SPN);
                __builtin_amdgcn_global_load_lds(vsrc, (lds_void*)&vst[64 * i], 16, 0, 0);
            }
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            __builtin_amdgcn_s_barrier();
            asm volatile("" ::: "memory");
            if constexpr (CONV) {
                // the entries' keys and values: conv outputs along the path, in place
                const int cs = tid >> 2, pt = tid & 3;
                if (cs < 16 || cs >= 32) {
                    for (int e = 0; e < ne; ++e) {
                        uint32_t* px = cs < 16 ? reinterpret_cast<uint32_t*>(&kst[e * 16 + cs]) + pt
                                               : reinterpret_cast<uint32_t*>(&reinterpret_cast<uint4*>(
                                                     recs[(cs - 32) >> 3])[8 * e + ((cs - 32) & 7)]) + pt;
                        const uint32_t xr = *px;
                        *px = conv2(tpp, hw0, hw1, hw2, xr);
                        hw0 = hw1;
                        hw1 = hw2;
                        hw2 = xr;
                    }
                }
                lds_barrier();
            }
            for (int e = 0; e < ne; ++e) {
                const float ae = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(pa), e));
                const float be = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(pb), e));
                float kf[kD / 32][8];
#pragma unroll
                for (int kb = 0; kb < kD / 32; ++kb) {
                    const uint4 w = kst[e * 16 + 4 * kb + (lane >> 4)];  // keys 32 kb + 8 (lane/16) ..
                    const uint32_t ww[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
                    for (int e2 = 0; e2 < 4; ++e2) {
                        kf[kb][2 * e2] = bf16_lo(ww[e2]);
                        kf[kb][2 * e2 + 1] = bf16_hi(ww[e2]);
                    }
                }
                float sk = 1.f;  // QKN: 1/|k| of the entry's key (every lane holds a quarter of it)
                if constexpr (QKN) {
                    float ss0 = 0.f, ss1 = 0.f;
#pragma unroll
                    for (int kb = 0; kb < kD / 32; ++kb)
#pragma unroll
                        for (int e8 = 0; e8 < 8; ++e8) {
                            float& acc = (kb & 1) ? ss1 : ss0;
                            acc = __builtin_fmaf(kf[kb][e8], kf[kb][e8], acc);
                        }
                    sk = __builtin_amdgcn_rsqf(row_group_sum(ss0 + ss1) + p.qk_eps);
                }
                float dl[NCT];
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) {
                    float s0 = 0.f, s1 = 0.f;
#pragma unroll
                    for (int kb = 0; kb < kD / 32; ++kb)
#pragma unroll
                        for (int e8 = 0; e8 < 8; ++e8) {
                            float& acc = (kb & 1) ? s1 : s0;
                            acc = __builtin_fmaf(__uint_as_float(raw[ct][kb][e8]), kf[kb][e8], acc);
                        }
                    const float u = row_group_sum(s0 + s1) * sk;
                    const float vj = bf16_lo((uint32_t)vsh[e * CW + NCT * (lane % 16) + ct]);
                    dl[ct] = be * __builtin_fmaf(-ae, u, vj) * sk;
                }
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
                    for (int kb = 0; kb < kD / 32; ++kb)
#pragma unroll
                        for (int e8 = 0; e8 < 8; ++e8)
                            raw[ct][kb][e8] = __float_as_uint(
                                __builtin_fmaf(dl[ct], kf[kb][e8], ae * __uint_as_float(raw[ct][kb][e8])));
            }
        }
        if constexpr (CONV) {  // this block's slice of the history (no other block reads it)
            *reinterpret_cast<uint32_t*>(hsl) = hn0;
            *reinterpret_cast<uint32_t*>(hsl + xc) = hn1;
            *reinterpret_cast<uint32_t*>(hsl + 2 * xc) = hn2;
            conv_cache_init(hn0, hn1, hn2);
        }
        float* Sw = pd.state + (((long)r * p.n_layers + l) * p.h_v + h) * (long)(kD * kD) +
                    (long)(8 * (lane / 16)) * kD + j0 + NCT * (lane % 16);
#pragma unroll
        for (int kb = 0; kb < kD / 32; ++kb)
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                if constexpr (NCT == 4)
                    *reinterpret_cast<uint4*>(Sw + (long)(32 * kb + e) * kD) =
                        make_uint4(raw[0][kb][e], raw[1][kb][e], raw[2][kb][e], raw[3][kb][e]);
                else
                    *reinterpret_cast<uint2*>(Sw + (long)(32 * kb + e) * kD) = make_uint2(raw[0][kb][e], raw[1][kb][e]);
            }
    };

    Rows rowC, rowA;  // this chunk, the next
    LaneInfo<D> info;
    if (!PEND || plen <= 0) {
        rowC = lane_rows(0);
        uint32_t h0 = 0, h1 = 0, h2 = 0;
        if constexpr (CONV) {  // the history of this thread's channels, as it is
            const uint16_t* hs = cf.hist + ((long)r * p.n_layers + l) * 3 * xc + walk_channel();
            h0 = *reinterpret_cast<const uint32_t*>(hs);
            h1 = *reinterpret_cast<const uint32_t*>(hs + xc);
            h2 = *reinterpret_cast<const uint32_t*>(hs + 2 * xc);
        }
        slab_load(0);
        slab_load(1);
        asm volatile("" ::: "memory");
        v_issue(rowC, vbufs[wave][0]);  // (its shuffles precede every copy)
        tile_issue(rowC);
        lane_info(0, rowC, info);
        rowA = N > kTile ? lane_rows(kTile) : rowC;
        slab_load(2);
        slab_load(3);
        if constexpr (CONV) conv_cache_init(h0, h1, h2);
    } else {
        if (N > 0) rowC = lane_rows(0);
#pragma unroll
        for (int kb = 0; kb < kD / 32; ++kb) slab_load(kb);
        // (Staging the first chunk's rows before the publication was measured slower: its
        // copies compete with the publication's.)
        pend_publish();
        if (N <= 0) return;  // uniform: nothing to verify for this request
        v_issue(rowC, vbufs[wave][0]);
        tile_issue(rowC);
        lane_info(0, rowC, info);
        rowA = N > kTile ? lane_rows(kTile) : rowC;
    }

    bf16x8 bhi[NCT][kD / 32], blo[NCT][kD / 32];
    // Each fp32 value x is held as hi + lo: hi = x truncated to bf16, lo = the exact
    // remainder x - hi rounded to nearest bf16 (|x - hi - lo| <= 2^-15 |x|).
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
        for (int kb = 0; kb < kD / 32; ++kb) {
            uint32_t hw[4], lw[4];
#pragma unroll
            for (int e2 = 0; e2 < 4; ++e2) {
                const uint32_t x0 = raw[ct][kb][2 * e2];
                const uint32_t x1 = raw[ct][kb][2 * e2 + 1];
                hw[e2] = __builtin_amdgcn_perm(x1, x0, 0x07060302u);  // {hi(x1), hi(x0)}: upper halves
                lw[e2] = f32x2_to_bf16x2(__uint_as_float(x0) - __uint_as_float(x0 & 0xffff0000u),
                                         __uint_as_float(x1) - __uint_as_float(x1 & 0xffff0000u));
            }
            bhi[ct][kb] = __builtin_bit_cast(bf16x8, make_uint4(hw[0], hw[1], hw[2], hw[3]));
            blo[ct][kb] = __builtin_bit_cast(bf16x8, make_uint4(lw[0], lw[1], lw[2], lw[3]));
        }

    // delta of the current path by depth; slot D takes the writes of nodes at depth D,
    // which have no descendants (their delta is never read)
    float dst[D + 1];
#pragma unroll
    for (int m = 0; m <= D; ++m) dst[m] = 0.f;
    // Gram tiles of this wave: rows = chunk keys (mt 0, Gram rows 16..47) or path-stack
    // keys (mt 1, Gram rows 0..15); columns = the chunk's keys (nt 0) or queries (nt 1)
    constexpr int NT = NW == 4 ? 1 : 2;
    const int mt = NW == 4 ? (wave >> 1) : wave;

    // R0 [k | q] of the 16 nodes of half hf of the chunk against the wave's CW columns,
    // then the 4 x 4 exchange of lane groups (permlane32, then permlane16 swaps) that
    // leaves lane l with column j0 + pc: pk[b][i], pq[b][i] belong to node 16 hf + 4 b + i.
    // CW = 32: pk holds the k products of tiles 0, 1 and then the q products of tiles
    // 0, 1 (pq is unused), so that after the exchange lane l < 32 holds R0 k and lane
    // l + 32 R0 q of the same column.
    auto half_products = [&](int hf, f32x4 (&pk)[4], f32x4 (&pq)[4]) {
#pragma unroll
        for (int ct = 0; ct < 4; ++ct)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                pk[ct][i] = 0.f;
                if constexpr (!AB) pq[ct][i] = 0.f;
            }
        const int nrow = 16 * hf + ln % 16;  // A rows: the half's nodes
#pragma unroll
        for (int kb = 0; kb < kD / 32; ++kb) {
            const int sw = (4 * kb + ln / 16) ^ (nrow & 15);
            const bf16x8 fk = as_bf16x8(tile.slot[nrow * 16 + sw]);
            const bf16x8 fq = as_bf16x8(tile.slot[(kTile + nrow) * 16 + sw]);
            if constexpr (AB) {
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) {
                    pk[ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fk, bhi[ct][kb], pk[ct], 0, 0, 0);
                    pk[ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fk, blo[ct][kb], pk[ct], 0, 0, 0);
                    pk[NCT + ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fq, bhi[ct][kb], pk[NCT + ct], 0, 0, 0);
                    pk[NCT + ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fq, blo[ct][kb], pk[NCT + ct], 0, 0, 0);
                }
                continue;
            }
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) {
                pk[ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fk, bhi[ct][kb], pk[ct], 0, 0, 0);
                pk[ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fk, blo[ct][kb], pk[ct], 0, 0, 0);
                pq[ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fq, bhi[ct][kb], pq[ct], 0, 0, 0);
                pq[ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fq, blo[ct][kb], pq[ct], 0, 0, 0);
            }
        }
    };
    // Lane group g holds tile ct as nodes 4 g + i of columns 16 ct + lane%16; after the
    // exchange lane group g holds, in block b, nodes 4 b + i of columns 16 g + lane%16.
    auto exchange = [&](f32x4 (&x)[4]) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int c = 0; c < 2; ++c) {
                const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(x[c][i]), __float_as_uint(x[c + 2][i]),
                                                                 false, false);
                x[c][i] = __uint_as_float(sw[0]);
                x[c + 2][i] = __uint_as_float(sw[1]);
            }
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int c = 0; c < 4; c += 2) {
                const auto sw = __builtin_amdgcn_permlane16_swap(__float_as_uint(x[c][i]), __float_as_uint(x[c + 1][i]),
                                                                 false, false);
                x[c][i] = __uint_as_float(sw[0]);
                x[c + 1][i] = __uint_as_float(sw[1]);
            }
    };

    for (int c0 = 0, buf = 0; c0 < N; c0 += kTile, buf ^= 1) {
        const bool more = c0 + kTile < N;
        const bool two = c0 + kTile / 2 < N;  // the second half holds real nodes
        Taps tp;
        if constexpr (CONV) load_taps(tp);  // lands with the chunk's copies
        // This chunk's tile, value rows and lane view have landed for every wave. The empty
        // asm consumes the lane view here, so that no first use of it later waits on the
        // copies issued below.
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        asm volatile("" ::"v"(info.dep), "v"(info.g), "v"(info.b), "v"(info.ci[0]), "v"(info.ci[D / 4 - 1]),
                     "v"(rowC.n), "v"(rowA.n), "v"(rowA.s));
        lds_barrier();
        if constexpr (CONV) {  // raw rows -> conv outputs, for every wave's rows
            conv_walk(tp, info);
            lds_barrier();
        }
        ln = lane;
        asm volatile("" : "+v"(ln));
        tn = ln % kTile;
        const int kb0 = ln / kTile;  // key block offset within a 16-key step (32x32x16 Gram)
        const int pc = NCT * (ln % 16) + (ln / 16) % NCT;  // this lane's state column (after the exchange)
        const int arow = mt == 0 ? tn : 2 * kTile + (tn & (kStack - 1));
        if constexpr (QKN) {
            // 1/sqrt(|x|^2 + eps) of every tile row: 8 lanes per row, 16 elements each
            for (int task = (int)threadIdx.x; task < kTileRows * 8; task += nthr) {
                const int row = task >> 3, grp = task & 7;
                const uint4 w0 = tile.slot[row * 16 + ((2 * grp) ^ (row & 15))];
                const uint4 w1 = tile.slot[row * 16 + ((2 * grp + 1) ^ (row & 15))];
                const uint32_t ww[8] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
                float ss = 0.f;
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    ss = __builtin_fmaf(bf16_lo(ww[i]), bf16_lo(ww[i]), ss);
                    ss = __builtin_fmaf(bf16_hi(ww[i]), bf16_hi(ww[i]), ss);
                }
                ss += __shfl_xor(ss, 1);
                ss += __shfl_xor(ss, 2);
                ss += __shfl_xor(ss, 4);
                if (grp == 0)
                    nrm[row < kTile ? kStack + row : row < 2 * kTile ? kCand + (row - kTile) : row - 2 * kTile] =
                        __builtin_amdgcn_rsqf(ss + p.qk_eps);
            }
        }
        if constexpr (!CONV) {
            if (c0 > 0) flush(vbufs[wave][buf ^ 1], kTile);  // the previous chunk had two halves
            if (more) {
                asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // the flush has read the buffer
                v_issue(rowA, vbufs[wave][buf ^ 1]);
            }
        }

        // ---- Gram (head-independent) into LDS
        {
            f32x16 gacc[NT];
#pragma unroll
            for (int i = 0; i < NT; ++i)
#pragma unroll
                for (int e = 0; e < 16; ++e) gacc[i][e] = 0.f;
#pragma unroll
            for (int s = 0; s < kD / 16; ++s) {
                const int sw = (2 * s + kb0) ^ (tn & 15);
                const bf16x8 fa = as_bf16x8(tile.slot[arow * 16 + sw]);
#pragma unroll
                for (int i = 0; i < NT; ++i) {
                    const int nt = NW == 4 ? (wave & 1) : i;
                    const bf16x8 fb = as_bf16x8(tile.slot[(nt * kTile + tn) * 16 + sw]);
                    gacc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa, fb, gacc[i], 0, 0, 0);
                }
            }
            // MFMA 32x32 output: lane holds column lane%32, rows 8(e/4) + 4(lane/32) + e%4
#pragma unroll
            for (int i = 0; i < NT; ++i) {
                const int nt = NW == 4 ? (wave & 1) : i;
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int row = 8 * (e / 4) + 4 * (ln / kTile) + e % 4;
                    if (mt == 0)
                        G[(kStack + row) * kGS + nt * kTile + tn] = gacc[i][e];
                    else if (e < 8)  // rows 0..15: the stack slots
                        G[row * kGS + nt * kTile + tn] = gacc[i][e];
                }
            }
        }
        f32x4 pk[4], pq[4];
        half_products(0, pk, pq);
        lds_barrier();  // the Gram is complete

        // ---- coefficient records of the wave's head (lanes 0..31: A, lanes 32..63: B);
        // with shared records the even wave of the head writes them
        if (rec_writer) {
            if (ln < kTile + kStack)
                walpha[ln < kTile ? kStack + ln : ln - kTile] =
                    __expf(rawg ? raw_log_alpha(info.g, alog, dtb) : info.g);
            const bool isB = ln >= kTile;
            const float* Gc = G + (isB ? kTile : 0) + tn;
            const float bt = rawg ? raw_beta(info.b) : info.b;
            float nk = 1.f, nq = 1.f;  // QKN: 1/|k_t|, 1/|q_t|
            if constexpr (QKN) {
                nk = nrm[kStack + tn];
                nq = nrm[kCand + tn];
            }
            const float sc = isB ? nq : bt * nk;
            float gam = walpha[kStack + tn];  // Gamma(a_{d-1} -> t) = alpha_t
            float cv[D];
#pragma unroll
            for (int m = D - 1; m >= 0; --m) {
                // ci is 0 past the depth: the reads stay in bounds and are masked, so they
                // are issued together instead of one conditional round trip per depth
                const bool live = m < info.dep;
                const int ci = live ? (int)((info.ci[m / 4] >> (8 * (m % 4))) & 0xffu) : 0;
                float gv = Gc[ci * kGS];
                if constexpr (QKN) gv *= nrm[ci];
                const float av = walpha[ci];
                cv[m] = (sc * gam) * gv * (live ? 1.f : 0.f);
                gam *= live ? av : 1.f;  // then Gamma(a_{m-1} -> t); finally gamma_t
            }
            float* rt = wrec + tn * W;
#pragma unroll
            for (int q4 = 0; q4 < D / 4; ++q4)
                *reinterpret_cast<float4*>(rt + 8 + (isB ? D : 0) + 4 * q4) =
                    make_float4(cv[4 * q4], cv[4 * q4 + 1], cv[4 * q4 + 2], cv[4 * q4 + 3]);
            if (!isB) {
                *reinterpret_cast<float4*>(rt) =
                    make_float4(__int_as_float(rowC.n), __int_as_float(info.dep), bt, gam * nk);
                *reinterpret_cast<float4*>(rt + 4) =
                    make_float4(G[(kStack + tn) * kGS + kTile + tn] * (nk * nq), gam * nq, 0.f, 0.f);
            }
        }
        // next chunk's lane view (lands during the recursion)
        Rows rowB = rowA;
        if (more) {
            lane_info(c0 + kTile, rowA, info);
            if (c0 + 2 * kTile < N) rowB = lane_rows(c0 + 2 * kTile);
        }
        if constexpr (SHR) lds_barrier();  // the head's records are written

        const float* rec = wrec;
        uint16_t* vs = reinterpret_cast<uint16_t*>(vbufs[wave][CONV ? 0 : buf]);
        // Straight-line over the 16 slots of a half: slots past the chunk's end hold exact
        // copies of its last node (tile rows, value row, record), so they recompute that
        // node's delta and output bit for bit and store the same value to the same place.
        // A node's record head: {row, depth, beta, gamma, k.q, gamma_q}, the first four
        // entries of A and B and the node's value entry. The next node's head is loaded
        // while the current node computes; the entries past the first four (nodes deeper
        // than 4) are loaded together, with one wait.
        struct RecHead {
            float4 w0, w1, a0, b0;  // w0 = {row, depth, beta, gamma}, w1 = {k.q, gamma_q, -, -}
            uint32_t vraw;
        };
        auto load_head = [&](int n, RecHead& h) {
            const float* cf = rec + n * W;
            h.w0 = *reinterpret_cast<const float4*>(cf);
            h.w1 = *reinterpret_cast<const float4*>(cf + 4);
            h.a0 = *reinterpret_cast<const float4*>(cf + 8);
            h.b0 = *reinterpret_cast<const float4*>(cf + 8 + D);
            h.vraw = vs[n * CW + pc];
        };
        auto recursion = [&](int hf, const f32x4 (&pk)[4], const f32x4 (&pq)[4]) {
            RecHead nx;
            load_head(16 * hf, nx);
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int n = 16 * hf + i;
                const RecHead cu = nx;
                if (i + 1 < 16) load_head(n + 1, nx);
                const int d = __builtin_amdgcn_readfirstlane(__float_as_int(cu.w0.y));  // uniform
                const float* cf = rec + n * W;
                // the entries 4 .. of A and B up to the node's depth (zero past it); with
                // D = 8 the four others are loaded with the head's wait, with D = 16 a group
                // at a time (registers)
                constexpr int kPre = D == 8 ? 1 : 0;  // groups loaded ahead of the sums
                float4 am[D / 4 > 1 ? D / 4 - 1 : 1], bm[D / 4 > 1 ? D / 4 - 1 : 1];
#pragma unroll
                for (int g = 1; g <= kPre; ++g) {
                    if (d > 4 * g) {  // uniform
                        am[g - 1] = *reinterpret_cast<const float4*>(cf + 8 + 4 * g);
                        bm[g - 1] = *reinterpret_cast<const float4*>(cf + 8 + D + 4 * g);
                    }
                }
                const float vj = __uint_as_float(cu.vraw << 16);
                // sums over the path stack as even/odd partial sums (half the dependent
                // chain), four depths at a time up to the node's depth: the record entries
                // past it are zero (the branch is uniform)
                float sa0 = __builtin_fmaf(cu.a0.x, dst[0], 0.f), sb0 = __builtin_fmaf(cu.b0.x, dst[0], 0.f);
                float sa1 = __builtin_fmaf(cu.a0.y, dst[1], 0.f), sb1 = __builtin_fmaf(cu.b0.y, dst[1], 0.f);
                sa0 = __builtin_fmaf(cu.a0.z, dst[2], sa0);
                sb0 = __builtin_fmaf(cu.b0.z, dst[2], sb0);
                sa1 = __builtin_fmaf(cu.a0.w, dst[3], sa1);
                sb1 = __builtin_fmaf(cu.b0.w, dst[3], sb1);
#pragma unroll
                for (int g = 1; g < D / 4; ++g) {
                    if (d <= 4 * g) break;
                    if (g > kPre) {
                        am[g - 1] = *reinterpret_cast<const float4*>(cf + 8 + 4 * g);
                        bm[g - 1] = *reinterpret_cast<const float4*>(cf + 8 + D + 4 * g);
                    }
                    sa0 = __builtin_fmaf(am[g - 1].x, dst[4 * g], sa0);
                    sb0 = __builtin_fmaf(bm[g - 1].x, dst[4 * g], sb0);
                    sa1 = __builtin_fmaf(am[g - 1].y, dst[4 * g + 1], sa1);
                    sb1 = __builtin_fmaf(bm[g - 1].y, dst[4 * g + 1], sb1);
                    sa0 = __builtin_fmaf(am[g - 1].z, dst[4 * g + 2], sa0);
                    sb0 = __builtin_fmaf(bm[g - 1].z, dst[4 * g + 2], sb0);
                    sa1 = __builtin_fmaf(am[g - 1].w, dst[4 * g + 3], sa1);
                    sb1 = __builtin_fmaf(bm[g - 1].w, dst[4 * g + 3], sb1);
                }
                const float gm = cu.w0.w, gq = QKN ? cu.w1.y : cu.w0.w;
                const float u = __builtin_fmaf(-gm, pk[i / 4][i % 4], vj);             // v - gamma R0 k
                const float delta = __builtin_fmaf(cu.w0.z, u, -(sa0 + sa1));          // beta u - sum A delta
                const float ov = __builtin_fmaf(cu.w1.x, delta, __builtin_fmaf(gq, pq[i / 4][i % 4], sb0 + sb1));
                dst[d < D ? d : D] = delta;            // uniform index: an indexed register write
                vs[n * CW + pc] = f32_to_bf16(ov);     // over the consumed value entry
            }
        };
        // CW = 32: lane l < 32 forms the sum over A and the delta of its column, lane
        // l + 32 the sum over B and the output, each from its own coefficient row; the
        // delta reaches the upper half with one permlane32 swap. The record (head and
        // every coefficient group) of the next node is loaded while the current one
        // computes.
        const bool hiB = ln >= kTile;
        struct RecHeadAB {
            float4 w0, w1, c[D / 4];
            uint32_t vraw;
        };
        auto load_head_ab = [&](int n, RecHeadAB& hd) {
            const float* cf = rec + n * W;
            hd.w0 = *reinterpret_cast<const float4*>(cf);
            hd.w1 = *reinterpret_cast<const float4*>(cf + 4);
#pragma unroll
            for (int g = 0; g < D / 4; ++g) hd.c[g] = *reinterpret_cast<const float4*>(cf + 8 + (hiB ? D : 0) + 4 * g);
            hd.vraw = vs[n * CW + pc];
        };
        // Each node starts by taking the record requested one node earlier into registers
        // and only then stores the previous node's output and requests the next record, so
        // its wait covers nothing issued since (the compiler's LDS waits here are full
        // drains, which would otherwise also wait for the record just requested).
        auto recursion_ab = [&](int hf, const f32x4 (&px)[4]) {
            RecHeadAB nx;
            load_head_ab(16 * hf, nx);
            uint16_t ovp = 0;  // the previous node's output, stored one node later
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int n = 16 * hf + i;
#pragma unroll
                for (int g = 0; g < D / 4; ++g)
                    asm volatile("" ::"v"(nx.c[g].x), "v"(nx.c[g].y), "v"(nx.c[g].z), "v"(nx.c[g].w));
                asm volatile("" ::"v"(nx.w0.y), "v"(nx.w0.z), "v"(nx.w0.w), "v"(nx.w1.x), "v"(nx.w1.y),
                             "v"(nx.vraw), "v"(ovp)
                             : "memory");
                if (i > 0 && hiB) vs[(n - 1) * CW + pc] = ovp;
                const RecHeadAB cu = nx;
                if (i + 1 < 16) load_head_ab(n + 1, nx);
                const int d = __builtin_amdgcn_readfirstlane(__float_as_int(cu.w0.y));  // uniform
                const float vj = __uint_as_float(cu.vraw << 16);
                // the partial sums of the 64-column form, over this lane's coefficients
                float s0 = __builtin_fmaf(cu.c[0].x, dst[0], 0.f);
                float s1 = __builtin_fmaf(cu.c[0].y, dst[1], 0.f);
                s0 = __builtin_fmaf(cu.c[0].z, dst[2], s0);
                s1 = __builtin_fmaf(cu.c[0].w, dst[3], s1);
#pragma unroll
                for (int g = 1; g < D / 4; ++g) {
                    if (d <= 4 * g) break;
                    s0 = __builtin_fmaf(cu.c[g].x, dst[4 * g], s0);
                    s1 = __builtin_fmaf(cu.c[g].y, dst[4 * g + 1], s1);
                    s0 = __builtin_fmaf(cu.c[g].z, dst[4 * g + 2], s0);
                    s1 = __builtin_fmaf(cu.c[g].w, dst[4 * g + 3], s1);
                }
                const float sm = s0 + s1;
                const float gm = cu.w0.w, gq = QKN ? cu.w1.y : cu.w0.w;
                // lower half: v - gamma R0 k; upper half: gamma_q R0 q + sum B delta
                const float t = __builtin_fmaf(hiB ? gq : -gm, px[i / 4][i % 4], hiB ? sm : vj);
                const float da = __builtin_fmaf(cu.w0.z, t, -sm);  // lower half: beta u - sum A delta
                const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(da), __float_as_uint(da), false, false);
                const float delta = __uint_as_float(sw[0]);  // the lower half's delta in both halves
                dst[d < D ? d : D] = delta;
                ovp = f32_to_bf16(__builtin_fmaf(cu.w1.x, delta, t));  // over the consumed value entry
            }
            if (hiB) vs[(16 * hf + 15) * CW + pc] = ovp;
        };
        exchange(pk);
        if constexpr (AB) {
            recursion_ab(0, pk);
        } else {
            exchange(pq);
            recursion(0, pk, pq);
        }
        if (two) half_products(1, pk, pq);
        lds_barrier();  // every wave has read the tile: it may be refilled
        if (more) tile_issue(rowA);
        if constexpr (CONV) {
            if (more) stack_from_cache();
        }
        if (two) {
            exchange(pk);
            if constexpr (AB) {
                recursion_ab(1, pk);
            } else {
                exchange(pq);
                recursion(1, pk, pq);
            }
        }
        if constexpr (CONV) {  // single value buffer: out, then the next chunk's rows in
            flush(vbufs[wave][0], two ? kTile : kTile / 2);
            if (more) {
                asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // the flush has read the buffer
                v_issue(rowA, vbufs[wave][0]);
            }
        }
        rowC = rowA;
        rowA = rowB;
    }
    if constexpr (!CONV) {  // the last chunk's outputs
        const int cl = (N - 1) / kTile;  // index of the last chunk
        flush(vbufs[wave][cl & 1], cl * kTile + kTile / 2 < N ? kTile : kTile / 2);
    }
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

}  // namespace lumo
