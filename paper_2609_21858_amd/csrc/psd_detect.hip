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
constexpr int kDetParts = 2;     // lanes per scored token (adjacent), each taking every other slot

template <int LAYOUT>
__global__ __launch_bounds__(kDetBlock) void detect_kernel(DetectArgs a) {
    __shared__ double part[kDetBlock / 64];
    __shared__ int cnt[kDetBlock / 64];
    const int i = blockIdx.x, tid = threadIdx.x, lane = tid & 63;
    const int sub = tid % kDetParts;
    const int32_t* toks = a.tokens + (size_t)i * a.seq_len;
    const int n0 = max(0, a.n0[i]);
    double acc = 0.0;
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
        const float tmin = fminf(emin, __shfl_xor(emin, 1));
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
        cmin = fmin(cmin, __shfl_xor(cmin, 1));
        if (sub == 0 && t < a.seq_len) {
            if (scored) {
                const double A = -log(-expm1(-(double)a.K * cmin));
                acc += A;
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
        acc += __shfl_xor(acc, off);
        c += __shfl_xor(c, off);
    }
    if (lane == 0) {
        part[tid >> 6] = acc;
        cnt[tid >> 6] = c;
    }
    __syncthreads();
    if (tid == 0) {
        double s = 0.0;
        int n = 0;
        for (int w = 0; w < kDetBlock / 64; ++w) {
            s += part[w];
            n += cnt[w];
        }
        a.out_score[i] = s;
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
        const double rs = mx + log(wave_sum_f64(lc == -INFINITY ? 0.0 : exp(lc - mx)));
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

// One wavefront per sequence (four per workgroup): ln p_A and ANLPPT_A of (S_A, M).
__global__ __launch_bounds__(256) void pvalue_kernel(int n, const double* score, const int32_t* count,
                                                      double* out_log_p, double* out_anlppt) {
    const int i = (int)(blockIdx.x * 4u + (threadIdx.x >> 6));
    if (i >= n) return;  // uniform per wavefront
    const double S = score[i];
    const int M = count[i];
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
    if ((threadIdx.x & 63) == 0) {
        out_log_p[i] = lp;
        if (out_anlppt) out_anlppt[i] = M > 0 ? -lp / (double)M : NAN;
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
    if (layout == 0)
        hipLaunchKernelGGL(detect_kernel<0>, dim3(a.n_seq), dim3(kDetBlock), 0, stream, a);
    else
        hipLaunchKernelGGL(detect_kernel<1>, dim3(a.n_seq), dim3(kDetBlock), 0, stream, a);
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
