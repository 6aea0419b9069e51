// Fused draft selection (Sec. V-D): one pass over a full-vocabulary logits row gives
// both the argmax (spine) token and the k ordered top-k candidates, each with its own
// tie rule, so the two reference outputs are reproduced without a second pass.
//
// Ranking. A logit maps to a 32-bit key whose unsigned order is the value order:
// NaN (any payload) above +inf, -0 equal to +0. A candidate is the 64-bit word
// (key << 32 | tie word): the tie word is the index itself when equal logits rank the
// higher index first, its complement when the lower index ranks first. All words of a
// row are distinct, so the top k are the k largest words. The spine is the largest
// (key << 32 | ~index): the lowest index among the maximal logits.
//
// Work split. A block streams one contiguous part of one row with 16-byte loads, a
// batch of kUnroll vectors per thread at a time. Each thread keeps its k largest words
// in registers, but only logits that can still matter reach that exact (integer)
// insertion: per batch the wave splits into G lane groups, takes each group's float
// maximum, and the k-th largest of those G maxima is a value that at least k logits
// seen by the wave reach; a logit strictly below it (float compare; NaN always passes,
// -0 equals +0) has k logits ranked above it and is skipped. Each wavefront then selects
// its k best words by k rounds of wave-wide maximum over the lanes' list heads (the
// winning lane pops its head; words are unique) and one more round for the spine word,
// and, when the block has the whole row, wave 0 does the same over the block's waves and
// writes the outputs. The cross-lane maxima use DPP moves and lane-row swaps, no LDS.
// When a row has several parts, each wavefront's words go to the workspace and a second
// kernel, one wavefront per row, merges them the same way; the kernel boundary orders
// the two, so nothing needs clearing between calls.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "device_common.h"
#include "lumo_tree.h"
#include "select.h"

namespace lumo {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kUnroll = 8;  // 16-byte loads in flight per thread (one batch)

__device__ __forceinline__ uint32_t rank_key(uint32_t u) {
    const uint32_t a = u & 0x7fffffffu;
    uint32_t key = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
    key = a == 0 ? 0x80000000u : key;
    return a > 0x7f800000u ? 0xffffffffu : key;
}

// Insert x into the descending list t (the smallest entry falls off the end).
template <int K>
__device__ __forceinline__ void topk_insert(uint64_t (&t)[K], uint64_t x) {
#pragma unroll
    for (int j = 0; j < K; ++j) {
        const uint64_t hi = t[j] > x ? t[j] : x;
        x = t[j] > x ? x : t[j];
        t[j] = hi;
    }
}

// Cross-lane moves without LDS: DPP within 16-lane rows, then the row-pair and
// half-wave swaps. DPP controls: quad permutations [1,0,3,2] and [2,3,0,1], mirror
// within 8-lane halves, mirror within the row.
constexpr int kDppXor1 = 0xB1, kDppXor2 = 0x4E, kDppHalfMirror = 0x141, kDppRowMirror = 0x140;

template <int CTRL>
__device__ __forceinline__ uint32_t dpp(uint32_t x) {
    return (uint32_t)__builtin_amdgcn_update_dpp((int)x, (int)x, CTRL, 0xF, 0xF, false);
}

template <int CTRL>
__device__ __forceinline__ uint64_t max_dpp(uint64_t x) {
    const uint64_t o = ((uint64_t)dpp<CTRL>((uint32_t)(x >> 32)) << 32) | dpp<CTRL>((uint32_t)x);
    return x > o ? x : o;
}

template <int CTRL>
__device__ __forceinline__ float fmax_dpp(float x) {
    return fmaxf(x, __uint_as_float(dpp<CTRL>(__float_as_uint(x))));
}

// Largest word of the wavefront, in every lane.
__device__ __forceinline__ uint64_t wave_max(uint64_t x) {
    x = max_dpp<kDppXor1>(x);
    x = max_dpp<kDppXor2>(x);
    x = max_dpp<kDppHalfMirror>(x);
    x = max_dpp<kDppRowMirror>(x);  // uniform within each 16-lane row
    const uint32_t lo = (uint32_t)x, hi = (uint32_t)(x >> 32);
    const auto l16 = __builtin_amdgcn_permlane16_swap(lo, lo, false, false);
    const auto h16 = __builtin_amdgcn_permlane16_swap(hi, hi, false, false);
    const uint64_t a = ((uint64_t)h16[0] << 32) | l16[0], b = ((uint64_t)h16[1] << 32) | l16[1];
    x = a > b ? a : b;  // rows 0-1 and rows 2-3
    const uint32_t lo2 = (uint32_t)x, hi2 = (uint32_t)(x >> 32);
    const auto l32 = __builtin_amdgcn_permlane32_swap(lo2, lo2, false, false);
    const auto h32 = __builtin_amdgcn_permlane32_swap(hi2, hi2, false, false);
    const uint64_t c = ((uint64_t)h32[0] << 32) | l32[0], d = ((uint64_t)h32[1] << 32) | l32[1];
    return c > d ? c : d;
}

// Pop the head of t if it is the round's winner (words are unique, so one thread does).
template <int K>
__device__ __forceinline__ void pop_if(uint64_t (&t)[K], uint64_t win) {
    if (win != 0 && t[0] == win) {
#pragma unroll
        for (int j = 0; j + 1 < K; ++j) t[j] = t[j + 1];
        t[K - 1] = 0;
    }
}

// The wavefront's k best words (out, descending; the lists are consumed) and its
// largest spine word, in every lane.
template <int K>
__device__ __forceinline__ void wave_select(uint64_t (&t)[K], uint64_t sp, uint64_t (&out)[K], uint64_t& spo) {
#pragma unroll
    for (int j = 0; j < K; ++j) {
        out[j] = wave_max(t[0]);
        pop_if<K>(t, out[j]);
    }
    spo = wave_max(sp);
}

// The block's k best words and spine word, valid in the lanes of wave 0.
template <int K>
__device__ __forceinline__ void block_select(uint64_t (&t)[K], uint64_t sp, uint64_t (&out)[K], uint64_t& spo,
                                             uint64_t (*red)[K + 1]) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    uint64_t w[K], wsp;
    wave_select<K>(t, sp, w, wsp);
    if (lane == 0) {
#pragma unroll
        for (int j = 0; j < K; ++j) red[wave][j] = w[j];
        red[wave][K] = wsp;
    }
    __syncthreads();
    if (wave != 0) return;
    // lane l < kWaves k holds word l % k of wave l / k; the rest hold nothing
    uint64_t c[1] = {lane < kWaves * K ? red[lane / K][lane % K] : 0};
    const uint64_t cs = lane < kWaves ? red[lane][K] : 0;
#pragma unroll
    for (int j = 0; j < K; ++j) {
        out[j] = wave_max(c[0]);
        pop_if<1>(c, out[j]);
    }
    spo = wave_max(cs);
}

template <int K>
__device__ __forceinline__ void write_result(const uint64_t (&t)[K], uint64_t sp, uint32_t tmask, long r,
                                             int32_t* __restrict__ spine, int32_t* __restrict__ cand) {
    spine[r] = (int32_t)~(uint32_t)sp;
#pragma unroll
    for (int j = 0; j < K; ++j) cand[r * K + j] = (int32_t)((uint32_t)t[j] ^ tmask);
}

// Element type traits: a 16-byte vector holds N logits; bits(i) is the float32 bit
// pattern of logit i of the vector; ninf is a vector word of -inf logits.
template <int DT>
struct Vec;
template <>
struct Vec<LUMO_F32> {
    static constexpr int N = 4;
    static constexpr uint32_t ninf = 0xff800000u;
    static __device__ __forceinline__ uint32_t bits(const uint4& w, int i) {
        return i == 0 ? w.x : i == 1 ? w.y : i == 2 ? w.z : w.w;
    }
    static __device__ __forceinline__ uint32_t one(const void* p, long e) {
        return static_cast<const uint32_t*>(p)[e];
    }
};
template <>
struct Vec<LUMO_BF16> {
    static constexpr int N = 8;
    static constexpr uint32_t ninf = 0xff80ff80u;
    static __device__ __forceinline__ uint32_t bits(const uint4& w, int i) {
        const uint32_t x = (i >> 1) == 0 ? w.x : (i >> 1) == 1 ? w.y : (i >> 1) == 2 ? w.z : w.w;
        return (i & 1) ? (x & 0xffff0000u) : (x << 16);
    }
    static __device__ __forceinline__ uint32_t one(const void* p, long e) {
        return ((uint32_t) static_cast<const uint16_t*>(p)[e]) << 16;
    }
};

template <int K, uint32_t TMASK>
__device__ __forceinline__ void take(uint64_t (&t)[K], uint64_t& sp, uint32_t bits, uint32_t idx) {
    const uint64_t hi = (uint64_t)rank_key(bits) << 32;
    topk_insert<K>(t, hi | (idx ^ TMASK));
    const uint64_t sw = hi | ~idx;
    sp = sp > sw ? sp : sw;
}

// Grid: rows x n_split blocks of kThreads; block b serves row b / n_split, part
// b % n_split. Vectors are 16-byte units counted from the (aligned) buffer start. The
// row's elements [r ld, r ld + vocab) cover the whole vectors [wa, wb), which the parts
// share evenly; the elements before wa and from wb on (fewer than N each, or the whole
// row when it has no whole vector) are read one by one by thread 0 of part 0.
template <int DT, int K, bool TIES_HIGH>
__global__ __launch_bounds__(kThreads) void select_part_kernel(const void* __restrict__ logits, int32_t vocab, long ld,
                                                               int32_t n_split, int32_t* __restrict__ spine,
                                                               int32_t* __restrict__ cand,
                                                               uint64_t* __restrict__ parts) {
    using V = Vec<DT>;
    constexpr int N = V::N;
    constexpr uint32_t tmask = TIES_HIGH ? 0u : 0xffffffffu;
    constexpr int G = K <= 4 ? 4 : 8;  // lane groups of the batch threshold
    constexpr int GL = 64 / G;
    __shared__ uint64_t red[kWaves][K + 1];

    const long r = blockIdx.x / n_split;
    const int s = blockIdx.x % n_split;
    const long rb = r * ld, re = rb + vocab;
    const long wa = (rb + N - 1) / N, wb = re / N;
    const long nw = wb > wa ? wb - wa : 0;
    const long chunk = (nw + n_split - 1) / n_split;
    const long p0 = wa + (long)s * chunk;
    const long p1 = min(p0 + chunk, wa + nw);

    uint64_t t[K];
#pragma unroll
    for (int j = 0; j < K; ++j) t[j] = 0;  // below every real word (min real key 0x007fffff)
    uint64_t sp = 0;
    float thr = -__builtin_inff();

    const uint4* vp = static_cast<const uint4*>(logits);
    for (long base = p0; base < p1; base += (long)kThreads * kUnroll) {
        uint4 w[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const long v = base + (long)u * kThreads + threadIdx.x;
            w[u] = v < p1 ? vp[v] : make_uint4(V::ninf, V::ninf, V::ninf, V::ninf);
        }
        // batch threshold: k-th largest of the lane groups' float maxima (NaN ignored
        // by fmaxf; a NaN logit passes the filter anyway)
        float m = -__builtin_inff();
#pragma unroll
        for (int u = 0; u < kUnroll; ++u)
#pragma unroll
            for (int i = 0; i < N; ++i) m = fmaxf(m, __uint_as_float(V::bits(w[u], i)));
        m = fmax_dpp<kDppXor1>(m);
        m = fmax_dpp<kDppXor2>(m);
        m = fmax_dpp<kDppHalfMirror>(m);  // uniform within 8-lane groups
        if (G == 4) m = fmax_dpp<kDppRowMirror>(m);  // within 16-lane groups
        float top[K];
#pragma unroll
        for (int j = 0; j < K; ++j) top[j] = -__builtin_inff();
#pragma unroll
        for (int q = 0; q < G; ++q) {
            float x = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(m), q * GL));
#pragma unroll
            for (int j = 0; j < K; ++j) {
                const float hi = fmaxf(top[j], x);
                x = fminf(top[j], x);
                top[j] = hi;
            }
        }
        thr = fmaxf(thr, top[K - 1]);
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const long v = base + (long)u * kThreads + threadIdx.x;
            if (v >= p1) continue;
#pragma unroll
            for (int i = 0; i < N; ++i) {
                const uint32_t b = V::bits(w[u], i);
                if (!(__uint_as_float(b) < thr)) take<K, tmask>(t, sp, b, (uint32_t)(v * N + i - rb));
            }
        }
    }
    if (s == 0 && threadIdx.x == 0) {  // partial vectors at the row's ends
        const long hend = nw > 0 ? wa * N : re, tbeg = nw > 0 ? wb * N : re;
        for (long e = rb; e < hend; ++e) take<K, tmask>(t, sp, V::one(logits, e), (uint32_t)(e - rb));
        for (long e = tbeg; e < re; ++e) take<K, tmask>(t, sp, V::one(logits, e), (uint32_t)(e - rb));
    }

    uint64_t best[K], bsp;
    if (n_split == 1) {  // the block has the whole row
        block_select<K>(t, sp, best, bsp, red);  // wave 0 holds the result
        if (threadIdx.x == 0) write_result<K>(best, bsp, tmask, r, spine, cand);
        return;
    }
    // each wavefront's words are one part of the row for the merge kernel
    wave_select<K>(t, sp, best, bsp);
    if ((threadIdx.x & 63) != 0) return;
    uint64_t* pp = parts + ((long)blockIdx.x * kWaves + (threadIdx.x >> 6)) * (K + 1);
#pragma unroll
    for (int j = 0; j < K; ++j) pp[j] = best[j];
    pp[K] = bsp;
}

// One wavefront per row: merge the row's n_parts parts ([K words, spine word] each).
template <int K, bool TIES_HIGH>
__global__ __launch_bounds__(64) void select_merge_kernel(int32_t n_parts, const uint64_t* __restrict__ parts,
                                                          int32_t* __restrict__ spine, int32_t* __restrict__ cand) {
    constexpr uint32_t tmask = TIES_HIGH ? 0u : 0xffffffffu;
    const long r = blockIdx.x;
    uint64_t t[K];
#pragma unroll
    for (int j = 0; j < K; ++j) t[j] = 0;
    uint64_t sp = 0;
    const uint64_t* rp = parts + r * n_parts * (K + 1);
    for (int p = threadIdx.x; p < n_parts; p += 64) {
        const uint64_t* pp = rp + (long)p * (K + 1);
#pragma unroll
        for (int j = 0; j < K; ++j) topk_insert<K>(t, pp[j]);
        sp = sp > pp[K] ? sp : pp[K];
    }
    uint64_t best[K];
    wave_select<K>(t, sp, best, sp);
    if (threadIdx.x == 0) write_result<K>(best, sp, tmask, r, spine, cand);
}

template <int DT, int K, bool TH>
hipError_t launch_kt(const SelectArgs& a, hipStream_t s) {
    const dim3 grid((unsigned)((long)a.rows * a.n_split)), block(kThreads);
    hipLaunchKernelGGL((select_part_kernel<DT, K, TH>), grid, block, 0, s, a.logits, a.vocab, a.ld, a.n_split, a.spine,
                       a.cand, a.parts);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || a.n_split == 1) return e;
    hipLaunchKernelGGL((select_merge_kernel<K, TH>), dim3((unsigned)a.rows), dim3(64), 0, s, a.n_split * kWaves,
                       a.parts, a.spine, a.cand);
    return hipGetLastError();
}

template <int DT, int K>
hipError_t launch_k(const SelectArgs& a, hipStream_t s) {
    return a.ties ? launch_kt<DT, K, true>(a, s) : launch_kt<DT, K, false>(a, s);
}

template <int DT>
hipError_t launch_dt(const SelectArgs& a, hipStream_t s) {
    switch (a.k) {
        case 1: return launch_k<DT, 1>(a, s);
        case 2: return launch_k<DT, 2>(a, s);
        case 3: return launch_k<DT, 3>(a, s);
        case 4: return launch_k<DT, 4>(a, s);
        case 5: return launch_k<DT, 5>(a, s);
        case 6: return launch_k<DT, 6>(a, s);
        case 7: return launch_k<DT, 7>(a, s);
        case 8: return launch_k<DT, 8>(a, s);
        default: return hipErrorNotSupported;
    }
}

}  // namespace

hipError_t launch_select(const SelectArgs& a, hipStream_t s) {
    if (a.rows == 0) return hipSuccess;
    return a.dtype == LUMO_BF16 ? launch_dt<LUMO_BF16>(a, s) : launch_dt<LUMO_F32>(a, s);
}

}  // namespace lumo
