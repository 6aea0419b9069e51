// Device helpers shared by the gfx950 kernels: operand decoding, the single
// per-value-row gated delta-rule update used by both verification and commit, and
// the XCD-aware block remap.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lumo {

// ---------------------------------------------------------------- bf16 / fp32 operands
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// fp32 -> bf16, round to nearest even (one v_cvt_pk_bf16_f32 on gfx950; NaN stays NaN).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// Two fp32 -> packed bf16 {lo: a, hi: b}, round to nearest even, one instruction.
__device__ __forceinline__ uint32_t f32x2_to_bf16x2(float a, float b) {
    const f32x2_t x = {a, b};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(x, bf16x2_t));
}

template <int OPT> struct Op;
template <> struct Op<0> {
    using T = float;
    static __device__ __forceinline__ float ld(const T* p, long i) { return p[i]; }
    static __device__ __forceinline__ void st(T* p, long i, float x) { p[i] = x; }
    // N consecutive values starting at p (N even, p 8-byte aligned)
    template <int N>
    static __device__ __forceinline__ void ld_row(const T* __restrict__ p, float (&out)[N]) {
#pragma unroll
        for (int i = 0; i < N; ++i) out[i] = p[i];
    }
};
template <> struct Op<1> {
    using T = uint16_t;
    static __device__ __forceinline__ float ld(const T* p, long i) { return __uint_as_float(((uint32_t)p[i]) << 16); }
    static __device__ __forceinline__ void st(T* p, long i, float x) { p[i] = f32_to_bf16(x); }
    template <int N>
    static __device__ __forceinline__ void ld_row(const T* __restrict__ p, float (&out)[N]) {
        const uint32_t* w = reinterpret_cast<const uint32_t*>(p);
#pragma unroll
        for (int i = 0; i < N / 2; ++i) {
            const uint32_t x = w[i];
            out[2 * i] = bf16_lo(x);
            out[2 * i + 1] = bf16_hi(x);
        }
    }
};

// ---------------------------------------------------------------- the recurrence
// Elements of k per uniform operand chunk (16 dwords of bf16: one scalar load).
constexpr int kChunk = 32;

// A wave-uniform offset hidden from the optimiser: every chunk of a key or query row
// is then loaded (scalar load) right where it is used instead of the whole row being
// hoisted and kept live; a wave holds about 100 scalar registers, fewer than one
// 128-wide fp32 row.
__device__ __forceinline__ int opaque(int x) {
    asm volatile("" : "+s"(x));
    return x;
}

// Dot product of a value row with a key or query row: element i goes into partial sum
// i % 4 (each in increasing i), then (s0 + s1) + (s2 + s3). Four independent chains
// instead of one of length d_k. Every kernel that applies the update uses this order,
// so verified and committed states agree bit for bit.
struct Dot4 {
    float s0 = 0.f, s1 = 0.f, s2 = 0.f, s3 = 0.f;
    __device__ __forceinline__ void add(int i, float a, float b) {  // i is a compile-time index
        switch (i & 3) {
            case 0: s0 = __builtin_fmaf(a, b, s0); break;
            case 1: s1 = __builtin_fmaf(a, b, s1); break;
            case 2: s2 = __builtin_fmaf(a, b, s2); break;
            default: s3 = __builtin_fmaf(a, b, s3); break;
        }
    }
    __device__ __forceinline__ float sum() const { return (s0 + s1) + (s2 + s3); }
};

// One gated delta-rule node update (Eq. (2)-(3)) for one value row j of the head
// matrix, S[i] = R[j][i]. `kp` is the node's key row (wave-uniform address, scalar
// loads chunk by chunk).
//   u = (R_pi k)_j;  delta = beta (v_j - alpha u);  R_j <- alpha R_j + delta k
// alpha is applied to the dot product instead of the matrix (same value in exact
// arithmetic). The operation order is fixed (explicit fma, contraction off), so
// verification and commit produce bitwise identical states. ks scales the key (1/|k|
// with query/key normalisation, else exactly 1, which leaves every value unchanged):
// delta = beta (v_j - alpha ks u) ks and R_j <- alpha R_j + delta k, the update with the
// normalised key.
template <int DK, int OPT>
__device__ __forceinline__ void gdn_row_update(float (&S)[DK], const typename Op<OPT>::T* __restrict__ kp,
                                               float vj, float alpha, float beta, float ks = 1.f) {
    constexpr int C = kChunk < DK ? kChunk : DK;
    Dot4 u;
#pragma unroll
    for (int c = 0; c < DK; c += C) {
        float kf[C];
        Op<OPT>::template ld_row<C>(kp + opaque(c), kf);
#pragma unroll
        for (int i = 0; i < C; ++i) u.add(c + i, S[c + i], kf[i]);
    }
    const float delta = beta * __builtin_fmaf(-alpha, u.sum() * ks, vj) * ks;
#pragma unroll
    for (int c = 0; c < DK; c += C) {
        float kf[C];
        Op<OPT>::template ld_row<C>(kp + opaque(c), kf);
#pragma unroll
        for (int i = 0; i < C; ++i) S[c + i] = __builtin_fmaf(delta, kf[i], alpha * S[c + i]);
    }
}

// o_j = (R_j . q) qs  (qs = 1/|q| with query/key normalisation, else exactly 1)
template <int DK, int OPT>
__device__ __forceinline__ float gdn_row_output(const float (&S)[DK], const typename Op<OPT>::T* __restrict__ qp,
                                                float qs = 1.f) {
    constexpr int C = kChunk < DK ? kChunk : DK;
    Dot4 o;
#pragma unroll
    for (int c = 0; c < DK; c += C) {
        float qf[C];
        Op<OPT>::template ld_row<C>(qp + opaque(c), qf);
#pragma unroll
        for (int i = 0; i < C; ++i) o.add(c + i, S[c + i], qf[i]);
    }
    return o.sum() * qs;
}

// 1/sqrt(|x|^2 + eps) of a wave-uniform query or key row (Sec. IV-B normalisation):
// one fma chain over the elements in index order, the order the commit's replay uses
// for its keys, so that prepared verification and prepared commit agree bit for bit.
template <int DK, int OPT>
__device__ __forceinline__ float row_rsq_norm(const typename Op<OPT>::T* __restrict__ xp, float eps) {
    constexpr int C = kChunk < DK ? kChunk : DK;
    float ss = 0.f;
#pragma unroll
    for (int c = 0; c < DK; c += C) {
        float xf[C];
        Op<OPT>::template ld_row<C>(xp + opaque(c), xf);
#pragma unroll
        for (int i = 0; i < C; ++i) ss = __builtin_fmaf(xf[i], xf[i], ss);
    }
    return __builtin_amdgcn_rsqf(ss + eps);
}

// ---------------------------------------------------------------- operand preparation
// Gates from raw inputs (Sec. IV-B; the Gated DeltaNet parametrisation):
//   log alpha = -exp(a_log) softplus(a + dt_bias),  softplus(x) = max(x, 0) + log(1 + e^-|x|)
//   beta = 1 / (1 + e^-b)
__device__ __forceinline__ float raw_log_alpha(float a, float a_log, float dt_bias) {
    const float x = a + dt_bias;
    const float sp = fmaxf(x, 0.f) + log1pf(__expf(-fabsf(x)));
    return -__expf(a_log) * sp;
}
__device__ __forceinline__ float raw_beta(float b) { return 1.f / (1.f + __expf(-b)); }

// ---------------------------------------------------------------- lane groups
// The sum of x over the four 16-lane rows of a wave, in every lane (the same bits in all
// four: (x0 + x1) + (x2 + x3)).
__device__ __forceinline__ float row_group_sum(float x) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    const float y = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(y), __float_as_uint(y), false, false);
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// ---------------------------------------------------------------- launch geometry
// Workgroups are dispatched round-robin over the 8 XCDs (each with its own L2).
// Remap so that consecutive logical block ids run on the same XCD: blocks that
// share operands (same segment and layer, neighbouring heads) then share an L2.
__device__ __forceinline__ int xcd_remap(int p, int nb) {
    constexpr int X = 8;
    const int xcd = p % X, local = p / X;
    const int base = nb / X, extra = nb % X;
    return (xcd < extra ? xcd * (base + 1) : extra * (base + 1) + (xcd - extra) * base) + local;
}

// Units of G consecutive logical blocks (blocks that share rows), each unit on one XCD
// and consecutive units on different XCDs: in every window of 8 G dispatched blocks,
// XCD x (blocks p = x mod 8) receives unit 8 w + x whole. Blocks of a last, partial
// window keep their order.
__device__ __forceinline__ int xcd_units(int p, int nb, int G) {
    constexpr int X = 8;
    const int win = X * G;
    if (p >= (nb / win) * win) return p;
    const int w = p / win, x = p % X, m = (p % win) / X;
    return (w * X + x) * G + m;
}

}  // namespace lumo
