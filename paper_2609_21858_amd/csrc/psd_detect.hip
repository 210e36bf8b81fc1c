// psd_detect.hip -- watermark detection score and parity exports (gfx950).
//
// Detection (eq. S_A; Alg. "Compute Aaronson score ..." in the appendix
// "Algorithm Implementation"): each scored token w_t recomputes its context key
// from the text alone (key, t, previous m tokens), rebuilds its K clocks
// E_j[w_t] exactly (float64), and adds A_t = -ln(1 - r_t) with
// r_t = exp(-K min_j E_j[w_t]) -- the target's clock of w_t in the augmented
// race is min_j E_j[w_t] ~ Exp(K), so r_t is uniform when the text does not
// carry the key.  One workgroup per sequence; the per-sequence sum runs in
// float64 in a fixed order (deterministic).
#include <hip/hip_runtime.h>

#include <math.h>

#include "psd_device.hpp"
#include "psd_launch.hpp"

namespace psd {

namespace {

template <int LAYOUT>
__global__ __launch_bounds__(kBlock) void detect_kernel(DetectArgs a) {
    __shared__ double part[kBlock];
    __shared__ int cnt[kBlock];
    const int i = blockIdx.x, tid = threadIdx.x;
    const int32_t* toks = a.tokens + (size_t)i * a.seq_len;
    const int n0 = max(0, a.n0[i]);
    double acc = 0.0;
    int c = 0;
    for (int t = tid; t < a.seq_len; t += kBlock) {
        const int w = toks[t];
        if (t < n0 || w < 0 || w >= a.V) {
            if (a.out_per_token) a.out_per_token[(size_t)i * a.seq_len + t] = NAN;
            continue;
        }
        int32_t win[16];
        for (int j = 0; j < a.m; ++j) {
            const int idx = t - a.m + j;
            win[j] = idx >= 0 ? toks[idx] : -1;
        }
        uint32_t k0, k1;
        context_key(a.key, t, win, a.m, k0, k1);
        double cmin = INFINITY;
        for (int j = 0; j < a.K; ++j) {
            const double e = LAYOUT == 0 ? tree_clock_f64((uint32_t)a.V, (uint32_t)j, (uint32_t)w, k0, k1)
                                         : flat_clock_f64((uint32_t)j, (uint32_t)w, k0, k1);
            cmin = fmin(cmin, e);
        }
        const double A = -log(-expm1(-(double)a.K * cmin));
        acc += A;
        ++c;
        if (a.out_per_token) a.out_per_token[(size_t)i * a.seq_len + t] = (float)A;
    }
    part[tid] = acc;
    cnt[tid] = c;
    __syncthreads();
    for (int s = kBlock / 2; s > 0; s >>= 1) {
        if (tid < s) {
            part[tid] += part[tid + s];
            cnt[tid] += cnt[tid + s];
        }
        __syncthreads();
    }
    if (tid == 0) {
        a.out_score[i] = part[0];
        a.out_count[i] = cnt[0];
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

__global__ void fill_zero_kernel(uint32_t* p, size_t n) {
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
        p[i] = 0u;
}

inline unsigned blocks_for(long n, int per) { return (unsigned)((n + per - 1) / per); }

}  // namespace

hipError_t launch_detect(const DetectArgs& a, int layout, hipStream_t stream) {
    if (a.n_seq <= 0) return hipSuccess;
    if (layout == 0)
        hipLaunchKernelGGL(detect_kernel<0>, dim3(a.n_seq), dim3(kBlock), 0, stream, a);
    else
        hipLaunchKernelGGL(detect_kernel<1>, dim3(a.n_seq), dim3(kBlock), 0, stream, a);
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
