// psd_detect.hip -- watermark detection score, its Gamma-tail p-value, and parity
// exports (gfx950).
//
// Detection (eq. S_A; Alg. "Compute Aaronson score ..." in the appendix
// "Algorithm Implementation"): each scored token w_t recomputes its context key
// from the text alone (key, t, previous m tokens), rebuilds its K clocks
// E_j[w_t] exactly (float64), and adds A_t = -ln(1 - r_t) with
// r_t = exp(-K min_j E_j[w_t]) -- the target's clock of w_t in the augmented
// race is min_j E_j[w_t] ~ Exp(K), so r_t is uniform when the text does not
// carry the key.  One workgroup of 1024 threads per sequence, two lanes per
// token (each rebuilds the token's context key and half of its K clocks).  The
// clocks are first computed in float to find the smallest; only slots whose float
// clock lies within a bound of float error of that minimum are rebuilt exactly in
// float64, so min_j E_j[w_t] is exact.  The per-sequence sum runs in float64 in a
// fixed order (deterministic).
#include <hip/hip_runtime.h>

#include <math.h>

#include "psd_device.hpp"
#include "psd_launch.hpp"

namespace psd {

namespace {

constexpr int kDetBlock = 1024;  // threads per detection workgroup
constexpr int kDetParts = 2;     // lanes per scored token (adjacent, a power of two), each taking
                                 // every kDetParts-th slot

// The further per-token scores of a pivot r = e^{-c}: the U-score r, Li et al.'s
// h*_{gum,Delta}(r) = log(k r^{Delta/(1-Delta)} + [q > 0] r^{(1-q)/q}) in log-sum-exp
// form, and Lattimore's min(eps^{-1/2}, (1 - r)^{-1/2}) - (2 - sqrt(eps)).
__device__ __forceinline__ double li_term(const DetectArgs& a, double c) {
    const double t1 = a.li_lnk - a.li_a * c;
    if (!a.li_q) return t1;
    const double t2 = -a.li_b * c;
    return fmax(t1, t2) + log1p(exp(-fabs(t1 - t2)));
}
__device__ __forceinline__ double pl_term(const DetectArgs& a, double c) {
    return fmin(a.pl_cap, 1.0 / sqrt(-expm1(-c))) - a.pl_c0;
}

template <int LAYOUT, bool MULTI>
__global__ __launch_bounds__(kDetBlock) void detect_kernel(DetectArgs a) {
    constexpr int NS = MULTI ? 4 : 1;
    __shared__ double part[NS][kDetBlock / 64];
    __shared__ int cnt[kDetBlock / 64];
    const int i = blockIdx.x, tid = threadIdx.x, lane = tid & 63;
    const int sub = tid % kDetParts;
    const int32_t* toks = a.tokens + (size_t)i * a.row_stride;
    const int n0 = max(0, a.n0[i]);
    double acc[NS];
#pragma unroll
    for (int q = 0; q < NS; ++q) acc[q] = 0.0;
    int c = 0;
    for (int t0 = 0; t0 < a.seq_len; t0 += kDetBlock / kDetParts) {
        // uniform trip count: both lanes of a token reach the shuffle
        const int t = t0 + tid / kDetParts;
        const int w = t < a.seq_len ? toks[t] : -1;
        const bool scored = t < a.seq_len && t >= n0 && w >= 0 && w < a.V;
        uint32_t k0 = 0u, k1 = 0u;
        float emin = INFINITY, e2 = INFINITY;  // this lane's smallest and second-smallest float clocks
        int jmin = -1;
        if (scored) {
            // context key: fold(key, t), then the m previous tokens oldest first (-1
            // before the text)
            k0 = (uint32_t)a.key;
            k1 = (uint32_t)(a.key >> 32);
            fold(k0, k1, (uint32_t)t, 0u, 0u);
            for (int j = 0; j < a.m; ++j) {
                const int idx = t - a.m + j;
                fold(k0, k1, (uint32_t)(idx >= 0 ? toks[idx] : -1), (uint32_t)j, 1u);
            }
            for (int j = sub; j < a.K; j += kDetParts) {
                const float e = LAYOUT == 0 ? tree_clock_f32((uint32_t)a.V, (uint32_t)j, (uint32_t)w, k0, k1)
                                            : flat_clock_f32((uint32_t)j, (uint32_t)w, k0, k1);
                if (e < emin) {
                    e2 = emin;
                    emin = e;
                    jmin = j;
                } else {
                    e2 = fminf(e2, e);
                }
            }
        }
        // Float clocks err by less than 1e-6 relative plus 1e-6 absolute (a few
        // roundings of positive terms, hardware log2); every slot within twice that
        // of the token's float minimum is rebuilt exactly.
        float tmin = emin;
#pragma unroll
        for (int o = 1; o < kDetParts; o <<= 1) tmin = fminf(tmin, __shfl_xor(tmin, o));
        const float lim = tmin + (tmin * 2e-6f + 2e-6f);
        double cmin = INFINITY;
        if (scored && emin <= lim) {
            if (e2 <= lim) {
                // another slot of this lane is close: rebuild all of them (rare)
                for (int j = sub; j < a.K; j += kDetParts)
                    cmin = fmin(cmin, LAYOUT == 0 ? tree_clock_f64((uint32_t)a.V, (uint32_t)j, (uint32_t)w, k0, k1)
                                                  : flat_clock_f64((uint32_t)j, (uint32_t)w, k0, k1));
            } else {
                cmin = LAYOUT == 0 ? tree_clock_f64((uint32_t)a.V, (uint32_t)jmin, (uint32_t)w, k0, k1)
                                   : flat_clock_f64((uint32_t)jmin, (uint32_t)w, k0, k1);
            }
        }
#pragma unroll
        for (int o = 1; o < kDetParts; o <<= 1) cmin = fmin(cmin, __shfl_xor(cmin, o));
        if (sub == 0 && t < a.seq_len) {
            if (scored) {
                const double cc = (double)a.K * cmin;  // the target's clock of w_t; pivot e^{-cc}
                const double A = -log(-expm1(-cc));
                acc[0] += A;
                if constexpr (MULTI) {
                    acc[1] += exp(-cc);
                    acc[2] += li_term(a, cc);
                    acc[3] += pl_term(a, cc);
                }
                ++c;
                if (a.out_per_token) a.out_per_token[(size_t)i * a.seq_len + t] = (float)A;
            } else if (a.out_per_token) {
                a.out_per_token[(size_t)i * a.seq_len + t] = NAN;
            }
        }
    }
    // fixed-order reduction: within each wave, then over the waves
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
#pragma unroll
        for (int q = 0; q < NS; ++q) acc[q] += __shfl_xor(acc[q], off);
        c += __shfl_xor(c, off);
    }
    if (lane == 0) {
#pragma unroll
        for (int q = 0; q < NS; ++q) part[q][tid >> 6] = acc[q];
        cnt[tid >> 6] = c;
    }
    __syncthreads();
    if (tid < NS) {
        double s = 0.0;
        for (int w = 0; w < kDetBlock / 64; ++w) s += part[tid][w];
        a.out_score[(size_t)i * NS + tid] = s;
    }
    if (tid == 0) {
        int n = 0;
        for (int w = 0; w < kDetBlock / 64; ++w) n += cnt[w];
        a.out_count[i] = n;
    }
}

__global__ void philox_kernel(int n, const uint32_t* ctr, const uint32_t* key, uint32_t* out) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const Words w = philox(ctr[4 * i], ctr[4 * i + 1], ctr[4 * i + 2], ctr[4 * i + 3], key[2 * i], key[2 * i + 1]);
    out[4 * i] = w.w0;
    out[4 * i + 1] = w.w1;
    out[4 * i + 2] = w.w2;
    out[4 * i + 3] = w.w3;
}

__global__ void context_keys_kernel(uint64_t key, int m, int n, const int64_t* t, const int32_t* windows,
                                    uint32_t* out) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    uint32_t k0, k1;
    context_key(key, t[i], windows + (size_t)i * m, m, k0, k1);
    out[2 * i] = k0;
    out[2 * i + 1] = k1;
}

__global__ void clock_values_kernel(int layout, int V, int n, const uint32_t* kappa, const int32_t* slot,
                                    const int32_t* token, double* out) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const uint32_t k0 = kappa[2 * i], k1 = kappa[2 * i + 1];
    const int v = token[i];
    if (v < 0 || v >= V) {
        out[i] = NAN;
        return;
    }
    out[i] = layout == 0 ? tree_clock_f64((uint32_t)V, (uint32_t)slot[i], (uint32_t)v, k0, k1)
                         : flat_clock_f64((uint32_t)slot[i], (uint32_t)v, k0, k1);
}

// ln Q(M, S), Q(M, S) = Gamma(M, S) / Gamma(M) the regularised upper incomplete gamma
// function, by one wavefront per sequence.  Both forms used are sums of positive
// terms that fall monotonically from their first term:
//  * S < M + 1: the power series of the lower function P = 1 - Q,
//    P = e^{-S} S^M / Gamma(M + 1) * sum_{n>=0} t_n, t_n = S^n / ((M+1)...(M+n))
//    (ratio S / (M + n) < 1), and ln Q = ln(1 - P);
//  * S >= M + 1: the Poisson form Q = sum_{k<M} e^{-S} S^k / k!, summed from
//    k = M - 1 down (ratio k / S < 1).
// A round gives each lane kTailChunk consecutive terms: the lane's first term in
// closed form (lgamma), the rest by the ratio, then a wave log-sum-exp.  Rounds
// stop once a round's last term is below e^-50 of the sum (the remaining tail is
// below that term times 1 / (1 - ratio) <~ sqrt(M) of it), or the terms run out.
constexpr int kTailChunk = 8;
constexpr int kTailTerms = 1 << 24;  // bound on the terms summed per sequence

__device__ __forceinline__ double wave_max_f64(double v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmax(v, __shfl_xor(v, o));
    return v;
}

__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    return v;
}

// ln of sum_n t_n (series: t_0 = 1; Poisson: the terms themselves).  Called by a
// whole wavefront with the same (S, M); `ok` is false if kTailTerms did not suffice.
__device__ double log_tail_sum(double S, int M, bool series, bool& ok) {
    const int lane = threadIdx.x & 63;
    const double a = (double)M, lnS = log(S), lg1 = lgamma(a + 1.0);
    double total = -INFINITY;
    ok = false;
    for (int base = 0; base < kTailTerms; base += 64 * kTailChunk) {
        const int n0 = base + lane * kTailChunk;
        const int k0 = M - 1 - n0;  // Poisson: the lane's first k
        double lt;                  // ln of the lane's first term
        if (series)
            lt = (double)n0 * lnS - (lgamma(a + (double)n0 + 1.0) - lg1);
        else
            lt = k0 >= 0 ? -S + (double)k0 * lnS - lgamma((double)k0 + 1.0) : -INFINITY;
        double t = 1.0, sum = 0.0;
        int j = 0;
        for (; j < kTailChunk; ++j) {
            const int n = n0 + j;
            if (!series && n > M - 1) break;
            if (j > 0) t *= series ? S / (a + (double)n) : (double)(M - n) / S;
            sum += t;
        }
        const double lc = sum > 0.0 ? lt + log(sum) : -INFINITY;
        const double mx = wave_max_f64(lc);
        if (mx == -INFINITY) {  // no term left (Poisson form exhausted)
            ok = true;
            break;
        }
        // (lane 0's sum for every lane: the butterfly's rounding may differ per lane, and
        // the stopping test below must be uniform)
        const double rs = mx + log(__shfl(wave_sum_f64(lc == -INFINITY ? 0.0 : exp(lc - mx)), 0));
        total = total == -INFINITY ? rs : fmax(total, rs) + log1p(exp(-fabs(total - rs)));
        // this round's last term (lane 63; -inf if its chunk ran past the last term)
        const double last = __shfl(j == kTailChunk ? lt + log(t) : -INFINITY, 63);
        if (last < total - 50.0) {
            ok = true;
            break;
        }
    }
    return total;
}

// ln p_A = ln Q(M, S) of one (S_A, M), by a whole wavefront.
__device__ double gamma_tail_log_p(double S, int M) {
    double lp;
    if (M < 0 || isnan(S)) {
        lp = NAN;
    } else if (M == 0 || S <= 0.0) {
        lp = 0.0;  // nothing scored, or no evidence: p = 1
    } else if (isinf(S)) {
        lp = -INFINITY;
    } else {
        const double a = (double)M;
        const bool series = S < a + 1.0;
        bool ok;
        const double ls = log_tail_sum(S, M, series, ok);
        lp = series ? log1p(-exp(-S + a * log(S) - lgamma(a + 1.0) + ls)) : ls;
        lp = ok ? fmin(lp, 0.0) : NAN;  // a probability: rounding above ln 1 is clamped
    }
    return lp;
}

// One wavefront per sequence (four per workgroup): ln p_A and ANLPPT_A of (S_A, M).
__global__ __launch_bounds__(256) void pvalue_kernel(int n, const double* score, const int32_t* count,
                                                      double* out_log_p, double* out_anlppt) {
    const int i = (int)(blockIdx.x * 4u + (threadIdx.x >> 6));
    if (i >= n) return;  // uniform per wavefront
    const double S = score[i];
    const int M = count[i];
    const double lp = gamma_tail_log_p(S, M);
    if ((threadIdx.x & 63) == 0) {
        out_log_p[i] = lp;
        if (out_anlppt) out_anlppt[i] = M > 0 ? -lp / (double)M : NAN;
    }
}

// ---- Chernoff bounds of the U-score and of Li et al.'s and Lattimore's scores:
// ln p <= min_{lam >= 0} M ln Phi(lam) - lam S, Phi(lam) = E[e^{lam h(U)}], U ~ Unif(0, 1)
// (App. "Gumbel Watermark" gives it for the U-score, Phi = (e^lam - 1) / lam).  The
// objective is convex with derivative M E_lam[h] - S (E_lam the tilted mean), so lam is
// found by bisection on that derivative.  Li and PL: Phi by composite 8-point
// Gauss-Legendre in the log domain, enough panels that each spans at most about one
// unit of the integrand's exponential rate:
//  * Li, with u = e^{-s}: Phi = int_0^inf e^{-s + lam L(s)} ds, L(s) = h(e^{-s}) =
//    logsumexp(ln k - a s, [q > 0] (-b s)); cut at s = 60 (the rest is below e^-59
//    of Phi), split where the faster of the two exponentials has died out;
//  * PL, with w = (1 - u)^{-1/2} on [1, eps^{-1/2}]: Phi = int 2 w^-3 e^{lam (w - c0)}
//    dw + eps e^{lam (eps^{-1/2} - c0)} (the truncated mass).
// 8-point Gauss-Legendre rule on [-1, 1] (Abramowitz & Stegun, Table 25.4).
__constant__ double kGLx[4] = {0.1834346424956498049394761, 0.5255324099163289858177390,
                               0.7966664774136267395915539, 0.9602898564975362316835609};
__constant__ double kGLw[4] = {0.3626837833783619829651504, 0.3137066458778872873379622,
                               0.2223810344533744705443560, 0.1012285362903762591525314};

// Online log-sum-exp of terms e^tau and of h e^tau.
struct LseAcc {
    double m, s, sh;
};
__device__ __forceinline__ void lse_add(LseAcc& A, double tau, double h) {
    if (tau == -INFINITY) return;
    if (tau > A.m) {
        const double f = exp(A.m - tau);
        A.s = A.s * f + 1.0;
        A.sh = A.sh * f + h;
        A.m = tau;
    } else {
        const double e = exp(tau - A.m);
        A.s += e;
        A.sh += h * e;
    }
}
__device__ __forceinline__ LseAcc lse_merge(LseAcc A, LseAcc B) {
    if (B.m == -INFINITY) return A;
    if (A.m == -INFINITY) return B;
    const double m = fmax(A.m, B.m), fa = exp(A.m - m), fb = exp(B.m - m);
    return LseAcc{m, A.s * fa + B.s * fb, A.sh * fa + B.sh * fb};
}
__device__ __forceinline__ LseAcc wave_lse(LseAcc A) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        const LseAcc B{__shfl_xor(A.m, o), __shfl_xor(A.s, o), __shfl_xor(A.sh, o)};
        A = lse_merge(A, B);
    }
    return A;
}

__device__ __forceinline__ double li_L(const ScorePvalueArgs& a, double s) {
    const double t1 = a.li_lnk - a.li_a * s;
    if (!a.li_q) return t1;
    const double t2 = -a.li_b * s;
    return fmax(t1, t2) + log1p(exp(-fabs(t1 - t2)));
}

// Composite Gauss-Legendre over [x0, x1] in n panels of the terms
// e^{ln(weight * jacobian) + exponent} (kind 2: Li in s, kind 3: PL in w), into A.
__device__ void gl_panels(const ScorePvalueArgs& a, int kind, double lam, double x0, double x1, int n, LseAcc& A) {
    const int lane = threadIdx.x & 63;
    const double w = (x1 - x0) / (double)n;
    for (int p = lane; p < n; p += 64) {
        const double mid = x0 + ((double)p + 0.5) * w, half = 0.5 * w;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const double x = mid + (j < 4 ? -kGLx[j] : kGLx[j - 4]) * half;
            const double lw = log(kGLw[j & 3] * half);
            double tau, h;
            if (kind == 2) {
                h = li_L(a, x);
                tau = lw - x + lam * h;
            } else {
                h = x - a.pl_c0;
                tau = lw + 0.69314718055994531 - 3.0 * log(x) + lam * h;
            }
            lse_add(A, tau, h);
        }
    }
}

// ln Phi(lam) and the tilted mean E_lam[h] of score kind 1 (U), 2 (Li), 3 (PL); whole wave.
__device__ void tilt(const ScorePvalueArgs& a, int kind, double lam, double& ln_phi, double& mean) {
    if (kind == 1) {
        if (lam < 1e-8) {
            ln_phi = 0.5 * lam;
            mean = 0.5 + lam / 12.0;
        } else {
            ln_phi = lam + log(-expm1(-lam)) - log(lam);
            mean = 1.0 / (-expm1(-lam)) - 1.0 / lam;
        }
        return;
    }
    LseAcc A{-INFINITY, 0.0, 0.0};
    constexpr int kMaxPanels = 16384;
    if (kind == 2) {
        const double cf = a.li_q ? fmax(a.li_a, a.li_b) : a.li_a;
        const double cs = a.li_q ? fmin(a.li_a, a.li_b) : a.li_a;
        const double s1 = cf > cs ? fmin(60.0, (fabs(a.li_lnk) + 40.0) / (cf - cs)) : 0.0;
        const int n1 = (int)fmin((double)kMaxPanels, ceil(s1 * (1.0 + lam * cf)) + 4.0);
        const int n2 = (int)fmin((double)kMaxPanels, ceil((60.0 - s1) * (1.0 + lam * cs)) + 4.0);
        if (s1 > 0.0) gl_panels(a, 2, lam, 0.0, s1, n1, A);
        gl_panels(a, 2, lam, s1, 60.0, n2, A);
    } else {
        const double W = a.pl_cap;
        if (W > 1.0) {
            const int n = (int)fmin((double)kMaxPanels, ceil((W - 1.0) * (lam + 3.0)) + 4.0);
            gl_panels(a, 3, lam, 1.0, W, n, A);
        }
        if ((threadIdx.x & 63) == 0) lse_add(A, log(a.pl_eps) + lam * (W - a.pl_c0), W - a.pl_c0);
    }
    A = wave_lse(A);
    // the butterfly combines the lanes' terms in a different order on each lane, so
    // results can differ in the last bit: every lane takes lane 0's, which keeps the
    // caller's bisection decisions (and with them every later shuffle) uniform
    ln_phi = __shfl(A.m + log(A.s), 0);
    mean = __shfl(A.sh / A.s, 0);
}

__device__ double chernoff_log_p(const ScorePvalueArgs& a, int kind, double S, int M) {
    if (M < 0 || isnan(S)) return NAN;
    if (M == 0) return 0.0;
    double lp0, mean0;
    tilt(a, kind, 0.0, lp0, mean0);
    if (S <= (double)M * mean0) return 0.0;
    double lo = 0.0, hi = 1.0, lnphi, mean;
    for (;;) {  // bracket the root of the derivative (doubling, at most 14 steps)
        tilt(a, kind, hi, lnphi, mean);
        if ((double)M * mean - S > 0.0 || hi >= 1e4) break;
        lo = hi;
        hi *= 2.0;
    }
    for (int it = 0; it < 100 && hi - lo > 1e-13 * hi; ++it) {
        const double mid = 0.5 * (lo + hi);
        tilt(a, kind, mid, lnphi, mean);
        if ((double)M * mean - S < 0.0)
            lo = mid;
        else
            hi = mid;
    }
    const double lam = 0.5 * (lo + hi);
    tilt(a, kind, lam, lnphi, mean);
    return fmin(0.0, (double)M * lnphi - lam * S);
}

// One wavefront per (sequence, score): ln p_A (exact Gamma tail) or a Chernoff bound.
__global__ __launch_bounds__(256) void score_pvalue_kernel(ScorePvalueArgs a) {
    const int item = (int)(blockIdx.x * 4u + (threadIdx.x >> 6));
    if (item >= 4 * a.n) return;  // uniform per wavefront
    const int i = item >> 2, kind = item & 3;
    const double S = a.scores[(size_t)i * 4 + kind];
    const int M = a.count[i];
    const double lp = kind == 0 ? gamma_tail_log_p(S, M) : chernoff_log_p(a, kind, S, M);
    if ((threadIdx.x & 63) == 0) a.out_log_p[(size_t)i * 4 + kind] = lp;
}

// Number of log p-values (stride apart) at or below ln alpha (NaN: not detected).
__global__ __launch_bounds__(1024) void detection_rate_kernel(int n, const double* log_p, int stride,
                                                               double log_alpha, int32_t* out) {
    __shared__ int part[16];
    int c = 0;
    for (int i = threadIdx.x; i < n; i += 1024) c += log_p[(size_t)i * stride] <= log_alpha ? 1 : 0;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) c += __shfl_xor(c, o);
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = c;
    __syncthreads();
    if (threadIdx.x == 0) {
        int t = 0;
        for (int w = 0; w < 16; ++w) t += part[w];
        *out = t;
    }
}

__global__ void fill_zero_kernel(uint32_t* p, size_t n) {
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
        p[i] = 0u;
}

inline unsigned blocks_for(long n, int per) { return (unsigned)((n + per - 1) / per); }

}  // namespace

hipError_t launch_detect(const DetectArgs& a, int layout, hipStream_t stream) {
    if (a.n_seq <= 0) return hipSuccess;
    if (a.multi) {
        if (layout == 0)
            hipLaunchKernelGGL((detect_kernel<0, true>), dim3(a.n_seq), dim3(kDetBlock), 0, stream, a);
        else
            hipLaunchKernelGGL((detect_kernel<1, true>), dim3(a.n_seq), dim3(kDetBlock), 0, stream, a);
    } else {
        if (layout == 0)
            hipLaunchKernelGGL((detect_kernel<0, false>), dim3(a.n_seq), dim3(kDetBlock), 0, stream, a);
        else
            hipLaunchKernelGGL((detect_kernel<1, false>), dim3(a.n_seq), dim3(kDetBlock), 0, stream, a);
    }
    return hipGetLastError();
}

hipError_t launch_score_pvalues(const ScorePvalueArgs& a, hipStream_t stream) {
    if (a.n <= 0) return hipSuccess;
    hipLaunchKernelGGL(score_pvalue_kernel, dim3(blocks_for((long)a.n * 4, 4)), dim3(256), 0, stream, a);
    return hipGetLastError();
}

hipError_t launch_detection_rate(int n, const double* log_p, int stride, double log_alpha, int32_t* out_count,
                                 hipStream_t stream) {
    hipLaunchKernelGGL(detection_rate_kernel, dim3(1), dim3(1024), 0, stream, n, log_p, stride, log_alpha, out_count);
    return hipGetLastError();
}

hipError_t launch_pvalue(int n, const double* score, const int32_t* count, double* out_log_p, double* out_anlppt,
                         hipStream_t stream) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(pvalue_kernel, dim3(blocks_for(n, 4)), dim3(256), 0, stream, n, score, count, out_log_p,
                       out_anlppt);
    return hipGetLastError();
}

hipError_t launch_philox(int n, const uint32_t* ctr, const uint32_t* key, uint32_t* out, hipStream_t stream) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(philox_kernel, dim3(blocks_for(n, 256)), dim3(256), 0, stream, n, ctr, key, out);
    return hipGetLastError();
}

hipError_t launch_context_keys(uint64_t key, int m, int n, const int64_t* t, const int32_t* windows,
                               uint32_t* out, hipStream_t stream) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(context_keys_kernel, dim3(blocks_for(n, 256)), dim3(256), 0, stream, key, m, n, t, windows,
                       out);
    return hipGetLastError();
}

hipError_t launch_clock_values(int layout, int V, int n, const uint32_t* kappa, const int32_t* slot,
                               const int32_t* token, double* out, hipStream_t stream) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(clock_values_kernel, dim3(blocks_for(n, 256)), dim3(256), 0, stream, layout, V, n, kappa,
                       slot, token, out);
    return hipGetLastError();
}

hipError_t launch_fill_zero(uint32_t* p, size_t n_words, hipStream_t stream) {
    if (n_words == 0) return hipSuccess;
    long blocks = (long)((n_words + 255) / 256);
    if (blocks > 4096) blocks = 4096;
    hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, p, n_words);
    return hipGetLastError();
}

}  // namespace psd
