// psd_device.hpp -- device building blocks of the keyed Poisson race on gfx950.
//
// Keyed randomness: Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11) keyed by a
// 64-bit context key kappa = H(key, t, last m tokens); the paper leaves the PRF
// open (Sec. 4.3: r_t(y) = F_{y_{t-m:t-1},k}(y); App. "Algorithm Implementation":
// Pi_t = G(k, Lambda(c_t))).  Clocks are iid Exp(1) per (slot, token) given kappa
// (eq. EFR), built by one of two layouts (see psd.h, psd_clocks).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace psd {

// ---------------------------------------------------------------- constants

constexpr uint32_t kPhiloxMulA = 0xD2511F53u;
constexpr uint32_t kPhiloxMulB = 0xCD9E8D57u;
constexpr uint32_t kPhiloxBumpA = 0x9E3779B9u;
constexpr uint32_t kPhiloxBumpB = 0xBB67AE85u;

// Counter word 3 tags the domain of a Philox call.
constexpr uint32_t kDomainFlat = 0u;  // flat clocks: ctr = (v >> 2, slot, 0, 0)
constexpr uint32_t kDomainKey = 1u;   // context-key fold
constexpr uint32_t kDomainTree = 2u;  // tree draws: ctr = (node, slot, level, 2) / (chunk, slot, 8 + half, 2)

// Token hierarchy of the tree layout: level L node i covers [i << kShift[L], ...).
// Level 1 = 8-token chunk, 2 = 128-token group, 3 = 2048, 4 = 32768, 5 = root.
constexpr int kShift1 = 3, kShift2 = 7, kShift3 = 11, kShift4 = 15, kShift5 = 19;
constexpr int kGroupTokens = 128;

// ln of the smallest clock value a flat word can produce: -ln(1 - 2^-24) = 5.9604645e-8,
// ln = -16.6355323.  Rounded down (a valid lower bound for every flat clock).
constexpr float kLnClockFloor = -16.6356f;

// ---------------------------------------------------------------- Philox

struct Words {
    uint32_t w0, w1, w2, w3;
};

__device__ __forceinline__ Words philox(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3, uint32_t k0,
                                        uint32_t k1) {
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        if (r) {
            k0 += kPhiloxBumpA;
            k1 += kPhiloxBumpB;
        }
        const uint64_t pa = (uint64_t)kPhiloxMulA * c0;
        const uint64_t pb = (uint64_t)kPhiloxMulB * c2;
        const uint32_t n0 = (uint32_t)(pb >> 32) ^ c1 ^ k0;
        const uint32_t n2 = (uint32_t)(pa >> 32) ^ c3 ^ k1;
        c1 = (uint32_t)pb;
        c3 = (uint32_t)pa;
        c0 = n0;
        c2 = n2;
    }
    return Words{c0, c1, c2, c3};
}

__device__ __forceinline__ uint32_t word_at(const Words& w, uint32_t i) {
    return i == 0 ? w.w0 : i == 1 ? w.w1 : i == 2 ? w.w2 : w.w3;
}

// ---------------------------------------------------------------- context key

// kappa_0 = fold(key, t), kappa_{i+1} = fold(kappa_i, w_i, i); fold = words 0, 1 of
// Philox(ctr = (a, b, tag, 1), kappa).
__device__ __forceinline__ void fold(uint32_t& k0, uint32_t& k1, uint32_t a, uint32_t b, uint32_t tag) {
    const Words w = philox(a, b, tag, kDomainKey, k0, k1);
    k0 = w.w0;
    k1 = w.w1;
}

__device__ __forceinline__ void context_key(uint64_t key, int64_t t, const int32_t* window, int m, uint32_t& k0,
                                            uint32_t& k1) {
    k0 = (uint32_t)key;
    k1 = (uint32_t)(key >> 32);
    const uint64_t tu = (uint64_t)t;
    fold(k0, k1, (uint32_t)tu, (uint32_t)(tu >> 32), 0u);
    for (int i = 0; i < m; ++i) fold(k0, k1, (uint32_t)window[i], (uint32_t)i, 1u);
}

// ---------------------------------------------------------------- uniforms

// U = (2 * (w >> 9) + 1) * 2^-24, exact in float and double.
__device__ __forceinline__ float uniform_f32(uint32_t w) { return (float)(2u * (w >> 9) + 1u) * 0x1p-24f; }
__device__ __forceinline__ double uniform_f64(uint32_t w) { return (double)(2u * (w >> 9) + 1u) * 0x1p-24; }

// E = -ln U.  The float version feeds pruning bounds only (hardware log2).
__device__ __forceinline__ float exp1_f32(uint32_t w) {
    return -__builtin_amdgcn_logf(uniform_f32(w)) * 0.69314718055994531f;
}
__device__ __forceinline__ double exp1_f64(uint32_t w) { return -log(uniform_f64(w)); }

__device__ __forceinline__ float ln_f32(float x) { return __builtin_amdgcn_logf(x) * 0.69314718055994531f; }

// e / n for a node of n tokens, with the hardware reciprocal: one rounding more than
// a division, and the float clocks only feed bounds that carry margins (the
// decisions and detection's minimum are rebuilt in float64).
__device__ __forceinline__ float div_n(float e, uint32_t n) { return e * __builtin_amdgcn_rcpf((float)n); }

// Uniform position in [0, n): floor(n * W / 2^64), W = (w1 << 32) | w2, exact integer arithmetic.
__device__ __forceinline__ uint32_t uniform_position(uint32_t w1, uint32_t w2, uint32_t n) {
    const uint64_t t = (uint64_t)w2 * n;
    const uint64_t u = (uint64_t)w1 * n + (t >> 32);
    return (uint32_t)(u >> 32);
}

// ---------------------------------------------------------------- tree draws

__device__ __forceinline__ uint32_t node_start(int shift, uint32_t i) { return i << shift; }
__device__ __forceinline__ uint32_t node_end(int shift, uint32_t i, uint32_t V) {
    const uint64_t e = ((uint64_t)i + 1u) << shift;
    return e < V ? (uint32_t)e : V;
}

// Minimum (m, p) of node (level, i) covering [cs, ce), given its parent's (m, p).
// Float version (pruning).
__device__ __forceinline__ void child_min_f32(float pm, uint32_t pp, int level, uint32_t i, uint32_t cs,
                                              uint32_t ce, uint32_t slot, uint32_t k0, uint32_t k1, float& m,
                                              uint32_t& p) {
    if (pp >= cs && pp < ce) {
        m = pm;
        p = pp;
        return;
    }
    const Words w = philox(i, slot, (uint32_t)level, kDomainTree, k0, k1);
    const uint32_t n = ce - cs;
    m = pm + div_n(exp1_f32(w.w0), n);
    p = cs + uniform_position(w.w1, w.w2, n);
}

__device__ __forceinline__ void child_min_f64(double pm, uint32_t pp, int level, uint32_t i, uint32_t cs,
                                              uint32_t ce, uint32_t slot, uint32_t k0, uint32_t k1, double& m,
                                              uint32_t& p) {
    if (pp >= cs && pp < ce) {
        m = pm;
        p = pp;
        return;
    }
    const Words w = philox(i, slot, (uint32_t)level, kDomainTree, k0, k1);
    const uint32_t n = ce - cs;
    m = pm + exp1_f64(w.w0) / (double)n;
    p = cs + uniform_position(w.w1, w.w2, n);
}

// Root minimum of a slot: Exp(1)/V at a uniform position.
__device__ __forceinline__ void root_min_f32(uint32_t V, uint32_t slot, uint32_t k0, uint32_t k1, float& m,
                                             uint32_t& p) {
    const Words w = philox(0u, slot, 5u, kDomainTree, k0, k1);
    m = div_n(exp1_f32(w.w0), V);
    p = uniform_position(w.w1, w.w2, V);
}

__device__ __forceinline__ void root_min_f64(uint32_t V, uint32_t slot, uint32_t k0, uint32_t k1, double& m,
                                             uint32_t& p) {
    const Words w = philox(0u, slot, 5u, kDomainTree, k0, k1);
    m = exp1_f64(w.w0) / (double)V;
    p = uniform_position(w.w1, w.w2, V);
}

// Exact clock of one token (tree layout), double: walk root -> token.  The six
// draws of the path (root, levels 4..1, token words) are independent Philox calls,
// issued together; the walk then uses a node's draw only where the parent's
// minimum lies outside it.
__device__ __forceinline__ double tree_clock_f64(uint32_t V, uint32_t slot, uint32_t v, uint32_t k0, uint32_t k1) {
    const int shifts[4] = {kShift4, kShift3, kShift2, kShift1};
    const Words wr = philox(0u, slot, 5u, kDomainTree, k0, k1);
    Words wn[4];
#pragma unroll
    for (int l = 0; l < 4; ++l) wn[l] = philox(v >> shifts[l], slot, (uint32_t)(4 - l), kDomainTree, k0, k1);
    const Words wt = philox(v >> 3, slot, 8u + ((v >> 2) & 1u), kDomainTree, k0, k1);
    double m = exp1_f64(wr.w0) / (double)V;
    uint32_t p = uniform_position(wr.w1, wr.w2, V);
#pragma unroll
    for (int l = 0; l < 4; ++l) {
        const int sh = shifts[l];
        const uint32_t i = v >> sh, cs = node_start(sh, i), ce = node_end(sh, i, V);
        if (!(p >= cs && p < ce)) {
            const uint32_t n = ce - cs;
            m = m + exp1_f64(wn[l].w0) / (double)n;
            p = cs + uniform_position(wn[l].w1, wn[l].w2, n);
        }
    }
    if (v == p) return m;
    return m + exp1_f64(word_at(wt, v & 3u));
}

// The same walk in float (hardware log2): relative error a few ulp plus an absolute
// error of about 2^-23 from logs of uniforms near 1; used to find the slot whose
// exact clock is smallest.
__device__ __forceinline__ float tree_clock_f32(uint32_t V, uint32_t slot, uint32_t v, uint32_t k0, uint32_t k1) {
    const int shifts[4] = {kShift4, kShift3, kShift2, kShift1};
    const Words wr = philox(0u, slot, 5u, kDomainTree, k0, k1);
    Words wn[4];
#pragma unroll
    for (int l = 0; l < 4; ++l) wn[l] = philox(v >> shifts[l], slot, (uint32_t)(4 - l), kDomainTree, k0, k1);
    const Words wt = philox(v >> 3, slot, 8u + ((v >> 2) & 1u), kDomainTree, k0, k1);
    float m = div_n(exp1_f32(wr.w0), V);
    uint32_t p = uniform_position(wr.w1, wr.w2, V);
#pragma unroll
    for (int l = 0; l < 4; ++l) {
        const int sh = shifts[l];
        const uint32_t i = v >> sh, cs = node_start(sh, i), ce = node_end(sh, i, V);
        if (!(p >= cs && p < ce)) {
            const uint32_t n = ce - cs;
            m = m + div_n(exp1_f32(wn[l].w0), n);
            p = cs + uniform_position(wn[l].w1, wn[l].w2, n);
        }
    }
    if (v == p) return m;
    return m + exp1_f32(word_at(wt, v & 3u));
}

__device__ __forceinline__ float flat_clock_f32(uint32_t slot, uint32_t v, uint32_t k0, uint32_t k1) {
    const Words w = philox(v >> 2, slot, 0u, kDomainFlat, k0, k1);
    return exp1_f32(word_at(w, v & 3u));
}

__device__ __forceinline__ double flat_clock_f64(uint32_t slot, uint32_t v, uint32_t k0, uint32_t k1) {
    const Words w = philox(v >> 2, slot, 0u, kDomainFlat, k0, k1);
    return exp1_f64(word_at(w, v & 3u));
}

// ---------------------------------------------------------------- lane reductions

// Max over each 16-lane DPP row; every lane of the row receives the result.
__device__ __forceinline__ float row16_max(float x) {
    int v = __float_as_int(x);
    x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(v, v, 0xB1, 0xF, 0xF, false)));  // quad [1,0,3,2]
    v = __float_as_int(x);
    x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(v, v, 0x4E, 0xF, 0xF, false)));  // quad [2,3,0,1]
    v = __float_as_int(x);
    x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(v, v, 0x141, 0xF, 0xF, false)));  // row_half_mirror
    v = __float_as_int(x);
    x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(v, v, 0x140, 0xF, 0xF, false)));  // row_mirror
    return x;
}

// Inclusive prefix sum over the 64 lanes of a wave (DPP: shifts within each row
// of 16 lanes, then row broadcasts of lanes 15 and 31).
__device__ __forceinline__ uint32_t wave_incl_sum(uint32_t v) {
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xF, 0xF, false);  // row_shr:1
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xF, 0xF, false);  // row_shr:2
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xF, 0xF, false);  // row_shr:4
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xF, 0xF, false);  // row_shr:8
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xA, 0xF, false);  // row_bcast:15 -> rows 1, 3
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xC, 0xF, false);  // row_bcast:31 -> rows 2, 3
    return v;
}

__device__ __forceinline__ float row16_min(float x) {
    int v = __float_as_int(x);
    x = fminf(x, __int_as_float(__builtin_amdgcn_update_dpp(v, v, 0xB1, 0xF, 0xF, false)));
    v = __float_as_int(x);
    x = fminf(x, __int_as_float(__builtin_amdgcn_update_dpp(v, v, 0x4E, 0xF, 0xF, false)));
    v = __float_as_int(x);
    x = fminf(x, __int_as_float(__builtin_amdgcn_update_dpp(v, v, 0x141, 0xF, 0xF, false)));
    v = __float_as_int(x);
    x = fminf(x, __int_as_float(__builtin_amdgcn_update_dpp(v, v, 0x140, 0xF, 0xF, false)));
    return x;
}

// Order-preserving map float -> int (for integer atomic min on scores).
__device__ __forceinline__ int ordered_key(float f) {
    const int i = __float_as_int(f);
    return i >= 0 ? i : i ^ 0x7FFFFFFF;
}
__device__ __forceinline__ float ordered_value(int k) { return __int_as_float(k >= 0 ? k : k ^ 0x7FFFFFFF); }

// bf16 -> f32 of the low / high half of a packed word.
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

}  // namespace psd
