// psd_gen.hip -- the multi-block generation loop on the device (gfx950).
//
// Speculative generation repeats one block per step (Alg. "Batched-target
// direct-top-k MPFR speculative sampling"; App. F's formal multi-draft algorithm):
// the models give the block's target and draft rows, the race and the walk emit
// tau tokens per sequence, and the emitted tokens extend every sequence's text, its
// next start position and its context window.  This file holds the device parts
// that the race does not: the commit of emitted tokens (advance_kernel) and a
// position-indexed toy language model standing in for the models (toy_rows_kernel),
// whose target row depends only on (sequence, absolute position) and whose drafter
// k adds its own noise -- so the emitted text must equal plain keyed decoding with
// the target rows, whatever the drafts (drafter invariance, App. C).
//
// Toy rows are exact functions of integer hashes (SplitMix64 per row, Wellons'
// lowbias32 per element) and of fp32 additions and products, each rounded once
// (no fused multiply-add), so any implementation of the same definition
// reproduces them bit for bit:
//   row words   R_T = sm(seed ^ sm(b << 32 | t)),  R_P = sm(R_T ^ 0xD1B54A32D192ED03),
//               R_D = sm(draft_seed ^ sm((k + 1) << 56 ^ b << 32 ^ t))   (sm = SplitMix64)
//   rank        r(v) = (a v + c) mod V,  c = R_P mod V,  a = (R_P >> 32) mod V moved up
//               to the next value coprime to V (a bijection of [0, V))
//   noise       x = lo32(R) + v * 0x9E3779B9 (mod 2^32), h = lowbias32(x);
//               target: 4 uniforms u = (q + 1/2) / 2^16 from the 16-bit halves of
//               h and of lowbias32(x ^ hi32(R_T)), n = (u1 + u2 + u3 + u4 - 2) * sqrt(3);
//               draft: n' = (u1 + u2 - 1) * sqrt(6) from the halves of h
//   rank term   q(r) = fp32(bits(fp32(1 + r)) - 0x3F800000), i.e. 2^23 times the
//               piecewise-linear log2 of 1 + r read off its fp32 bits, and the weight
//               w = fp32(-alpha ln 2 / 2^23) (computed in double), so w q(r) is close
//               to -alpha ln(1 + r): a Zipf-like head
//   logits      z_v = sigma * n + w * q(r(v)),  draft_v = z_v + tau_b * n'
//               (tau_b = tau[0] for b < tau_split, else tau[1]); bf16 rows are the
//               round-to-nearest-even of those fp32 values.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "psd_launch.hpp"

// The toy rows' definition rounds every product and sum once: no contraction into
// fused multiply-adds anywhere in this file (the build passes -ffp-contract=off too).
#pragma clang fp contract(off)

namespace psd {

namespace {

__device__ __forceinline__ uint64_t sm64(uint64_t x) {
    x += 0x9E3779B97F4A7C15ull;
    x = (x ^ (x >> 30)) * 0xBF58476D1CE4E5B9ull;
    x = (x ^ (x >> 27)) * 0x94D049BB133111EBull;
    return x ^ (x >> 31);
}

__device__ __forceinline__ uint32_t lowbias32(uint32_t x) {
    x ^= x >> 16;
    x *= 0x7FEB352Du;
    x ^= x >> 15;
    x *= 0x846CA68Bu;
    x ^= x >> 16;
    return x;
}

__device__ __forceinline__ uint32_t gcd32(uint32_t a, uint32_t b) {
    while (b) {
        const uint32_t t = a % b;
        a = b;
        b = t;
    }
    return a;
}

// Sum of the two (q + 1/2) / 2^16 uniforms held in the halves of h (exact in fp32).
__device__ __forceinline__ float two_uniforms(uint32_t h) {
    return ((float)(h & 0xFFFFu) + (float)(h >> 16) + 1.0f) * 0x1p-16f;
}

__device__ __forceinline__ uint16_t bf16_rne(float f) {
    const uint32_t u = __float_as_uint(f);
    return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

// One workgroup per (sequence b, depth s): the target row at t = start[b] + s and,
// for s < gamma, the K draft rows of that depth.
template <bool BF16>
__global__ __launch_bounds__(256) void toy_rows_kernel(ToyArgs a) {
    const int G1 = a.gamma + 1;
    const int b = blockIdx.x / G1, s = blockIdx.x % G1;
    const uint64_t t = (uint64_t)(a.start_pos[b] + s);
    const uint32_t V = (uint32_t)a.V;
    const uint64_t RT = sm64(a.seed ^ sm64(((uint64_t)b << 32) | (t & 0xFFFFFFFFull)));
    const uint64_t RP = sm64(RT ^ 0xD1B54A32D192ED03ull);
    const uint32_t c = (uint32_t)(RP % V);
    uint32_t am = (uint32_t)((RP >> 32) % V);
    if (am == 0u) am = 1u;
    while (gcd32(am, V) != 1u) am = am + 1u == V ? 1u : am + 1u;
    const float tau = b < a.tau_split ? a.tau0 : a.tau1;
    const bool drafts = s < a.gamma && a.draft_logits;
    __shared__ uint32_t rd[32];  // lo32(R_D) of each drafter at this (b, t)
    if ((int)threadIdx.x < a.K)
        rd[threadIdx.x] = (uint32_t)sm64(a.draft_seed ^ sm64(((uint64_t)(threadIdx.x + 1) << 56) ^
                                                             ((uint64_t)b << 32) ^ (t & 0xFFFFFFFFull)));
    __syncthreads();
    const size_t trow = ((size_t)b * G1 + s) * V;
    // r(v) stepped along this thread's stride: r(v + stride) = r(v) + a * stride (mod V)
    uint32_t r = (uint32_t)(((uint64_t)am * threadIdx.x + c) % V);
    const uint32_t step = (uint32_t)(((uint64_t)am * blockDim.x) % V);
    for (uint32_t v = threadIdx.x; v < V; v += blockDim.x) {
        const uint32_t x = (uint32_t)RT + v * 0x9E3779B9u;
        const float u4 = two_uniforms(lowbias32(x)) + two_uniforms(lowbias32(x ^ (uint32_t)(RT >> 32)));
        const float n = __fmul_rn(u4 - 2.0f, 1.7320508075688772f);
        const float q = (float)(int32_t)(__float_as_uint((float)(r + 1u)) - 0x3F800000u);
        const float z = __fadd_rn(__fmul_rn(a.sigma, n), __fmul_rn(a.w, q));
        r += step;
        if (r >= V) r -= V;
        if (BF16)
            ((uint16_t*)a.target_logits)[trow + v] = bf16_rne(z);
        else
            ((float*)a.target_logits)[trow + v] = z;
        if (!drafts) continue;
        for (int k = 0; k < a.K; ++k) {
            const float n2 = __fmul_rn(two_uniforms(lowbias32(rd[k] + v * 0x9E3779B9u)) - 1.0f, 2.449489742783178f);
            const float d = __fadd_rn(z, __fmul_rn(tau, n2));
            const size_t drow = (((size_t)b * a.K + k) * a.gamma + s) * V;
            if (BF16)
                ((uint16_t*)a.draft_logits)[drow + v] = bf16_rne(d);
            else
                ((float*)a.draft_logits)[drow + v] = d;
        }
    }
}

constexpr int kAdvBlock = 1024;

// Commit the emitted tokens of one block (or, with out_len NULL, set up the first
// block from the prompt), then the next block's start positions and windows and the
// number of sequences still short of max_len.  One workgroup, sequences strided.
__global__ __launch_bounds__(kAdvBlock) void advance_kernel(AdvanceArgs a) {
    __shared__ int red[kAdvBlock / 64];
    const int tid = threadIdx.x;
    int active = 0;
    for (int b = tid; b < a.B; b += kAdvBlock) {
        int32_t* text = a.text + (size_t)b * a.text_stride;
        int64_t L = a.out_len ? a.length[b] : (int64_t)a.m;
        L = L < a.m ? a.m : (L > a.max_len ? a.max_len : L);  // keeps every index below in range
        if (a.out_len && L < a.max_len) {
            const int n = min(max(a.out_len[b], 0), a.gamma + 1);
            for (int i = 0; i < n && L < a.max_len; ++i) {
                const int32_t y = a.out_tokens[(size_t)b * (a.gamma + 1) + i];
                if (y < 0) {  // an empty row: the sequence cannot continue
                    for (; L < a.max_len; ++L) text[L] = -1;
                    break;
                }
                text[L++] = y;
            }
        }
        a.length[b] = L;
        const int64_t st = L < a.max_len ? L : a.max_len - 1;
        a.start_pos[b] = st;
        for (int i = 0; i < a.m; ++i) a.prefix[(size_t)b * a.m + i] = text[st - a.m + i];
        active += L < a.max_len;
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) active += __shfl_xor(active, o);
    if ((tid & 63) == 0) red[tid >> 6] = active;
    __syncthreads();
    if (tid == 0) {
        int total = 0;
        for (int w = 0; w < kAdvBlock / 64; ++w) total += red[w];
        *a.n_active = total;
    }
}

}  // namespace

hipError_t launch_toy_rows(const ToyArgs& a, bool bf16, hipStream_t stream) {
    const long blocks = (long)a.B * (a.gamma + 1);
    if (blocks <= 0) return hipSuccess;
    if (bf16)
        hipLaunchKernelGGL(toy_rows_kernel<true>, dim3((unsigned)blocks), dim3(256), 0, stream, a);
    else
        hipLaunchKernelGGL(toy_rows_kernel<false>, dim3((unsigned)blocks), dim3(256), 0, stream, a);
    return hipGetLastError();
}

hipError_t launch_advance(const AdvanceArgs& a, hipStream_t stream) {
    hipLaunchKernelGGL(advance_kernel, dim3(1), dim3(kAdvBlock), 0, stream, a);
    return hipGetLastError();
}

}  // namespace psd
