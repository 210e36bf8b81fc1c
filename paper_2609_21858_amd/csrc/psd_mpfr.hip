// psd_mpfr.hip -- drafting with identical drafters: multi-sample PFR (gfx950).
//
// Sec. 5 (eq. MPFR) with the direct finite-support sampler of the appendix "A
// better finite-support MPFR implementation": token v's unit-rate clock has
// arrivals G_{v,j} = E_0[v] + ... + E_j[v] (slot i of the keyed source is v's
// (i+1)-th exponential), and the nu samples of a context are the labels of the nu
// smallest ln G_{v,j} - l_v / T over (v, j < nu).  In Alg. "Multi-Draft ...
// (Formal)" the K drafts of a block form a context tree with multiplicities; here
// the tree is held as K paths: at depth s the paths with equal drafts so far share
// one context, whose proposal row is its lowest path's row, and the context's i-th
// sample goes to its i-th path.
//
// One workgroup per draft row (b, k) of a depth.  Either every workgroup streams
// its row once (log-sum-exp, maxima of 128-token groups), one launch per depth, or
// a streaming launch has done so for every row of the call; then one launch can run
// every depth, each workgroup going on to the next depth as soon as the drafts its
// context depends on have landed.  The workgroup of a context's lowest path samples
// the context:
//  1. seeds: the largest token of the top group of each eighth of the row; their
//     first nu arrivals, exact in fp64, give theta = the nu-th smallest of those
//     scores, an upper bound on the context's nu-th smallest score;
//  2. since G_{v,j} >= E_0[v], every token of a sample has a slot-0 score at most
//     theta: a descent of slot 0's tree (root, 32768-, 2048- and 128-token nodes,
//     8-token chunks) lists every token whose slot-0 score, in fp32 with a margin,
//     is at most theta (flat clocks: every group whose clock-floor bound passes);
//  3. the listed tokens' arrivals are rebuilt exactly in fp64 one at a time, and nu
//     rounds of a workgroup-wide lexicographic minimum over (score, token, arrival)
//     emit the samples in order (exact ties: lowest token, then lowest arrival).
// The fp32 scores use (l - row maximum) / T, like the race kernel.
#include <hip/hip_runtime.h>

#include <math.h>

#include "psd_device.hpp"
#include "psd_launch.hpp"
#include "psd_layout.hpp"

namespace psd {

namespace {

constexpr int kMBlock = 256;
constexpr int kMaxGroups = 4096;  // 128-token groups of V <= 2^19
constexpr int kMCand = 1024;      // listed candidate tokens of a context
constexpr int kSeeds = 8;
static_assert(kSeeds == 8, "the workspace holds 8 seed tokens per streamed row");
constexpr float kMMargin = 1e-3f;  // fp32 pruning margin (score units)
constexpr uint32_t kMErrCand = 2u;

struct MNode {
    uint32_t i;  // node index at its level
    float m;     // slot-0 minimum clock of the node
    uint32_t p;  // token holding it
};

struct MShared {
    float m3[256];             // 2048-token block maxima
    float m4[16];              // 32768-token node maxima
    int seed_g[kSeeds];
    int seed_tok[kSeeds];
    double pair[kSeeds * 32];  // seed arrival scores (shifted frame)
    MNode l4[16];
    MNode l3[256];
    MNode lg[256];             // surviving groups of one batch of level-3 nodes
    int cand_v[kMCand];
    float cand_x[kMCand];
    int cand_j[kMCand];
    union {
        int path_tok[32 * 32];  // draft tokens of the K paths at depths < s ([path][depth]):
                                // read up to the context key only
        double cand_g[kMCand];  // the listed tokens' cumulative clocks (arrival phase)
    };
    double cand_s[kMCand];
    float red_m[kMBlock / 64], red_s[kMBlock / 64], red_x[kMBlock / 64];
    double red_d[kMBlock / 64];
    int red_v[kMBlock / 64], red_j[kMBlock / 64], red_i[kMBlock / 64];
    uint32_t mask;
    int n_l4, n_l3, n_lg, n_cand;
    float rowmax, theta;
    uint32_t kappa0, kappa1;
    int samples[32];
    int pre[16];               // the sequence's context window before the block (m <= 16)
    uint32_t epoch;            // this launch's tag of the handed-over drafts (multi-depth launch)
};

__device__ __forceinline__ float mload(const unsigned char* row, bool bf16, int v) {
    return bf16 ? __uint_as_float((uint32_t)((const uint16_t*)row)[v] << 16) : ((const float*)row)[v];
}

// 8 logits from `base` (-inf past V).
template <bool BF16, bool VEC>
__device__ __forceinline__ void mload8(const unsigned char* row, int V, int base, float (&x)[8]) {
    if constexpr (VEC) {
        if constexpr (BF16) {
            uint4 u = make_uint4(0xFF80FF80u, 0xFF80FF80u, 0xFF80FF80u, 0xFF80FF80u);
            if (base < V) u = *(const uint4*)((const uint16_t*)row + base);
            x[0] = bf16_lo(u.x); x[1] = bf16_hi(u.x); x[2] = bf16_lo(u.y); x[3] = bf16_hi(u.y);
            x[4] = bf16_lo(u.z); x[5] = bf16_hi(u.z); x[6] = bf16_lo(u.w); x[7] = bf16_hi(u.w);
        } else {
            float4 f0 = make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY), f1 = f0;
            if (base < V) f0 = *(const float4*)((const float*)row + base);
            if (base + 4 < V) f1 = *(const float4*)((const float*)row + base + 4);
            x[0] = f0.x; x[1] = f0.y; x[2] = f0.z; x[3] = f0.w;
            x[4] = f1.x; x[5] = f1.y; x[6] = f1.z; x[7] = f1.w;
        }
    } else {
#pragma unroll
        for (int i = 0; i < 8; ++i) x[i] = base + i < V ? mload(row, BF16, base + i) : -INFINITY;
    }
}

// Raw words of 8 logits for a load issued ahead of its use (vector path: one or two
// 16-byte loads, the address clamped into the row; scalar path: nothing loaded ahead).
template <bool BF16, bool VEC>
struct MRaw {
    uint4 w[BF16 ? 1 : 2];
};
template <bool BF16, bool VEC>
__device__ __forceinline__ void mraw_load(const unsigned char* row, int V, int base, MRaw<BF16, VEC>& r) {
    if constexpr (VEC) {
        if constexpr (BF16) {
            r.w[0] = *(const uint4*)((const uint16_t*)row + min(base, V - 8));
        } else {
            r.w[0] = *(const uint4*)((const float*)row + min(base, V - 4));
            r.w[1] = *(const uint4*)((const float*)row + min(base + 4, V - 4));
        }
    }
}
// The 8 logits from `base` (-inf past V) out of the raw words (scalar path: loaded here).
template <bool BF16, bool VEC>
__device__ __forceinline__ void mraw_unpack(const unsigned char* row, int V, int base, const MRaw<BF16, VEC>& r,
                                            float (&x)[8]) {
    if constexpr (VEC) {
        if constexpr (BF16) {
            const uint4 u = r.w[0];
            x[0] = bf16_lo(u.x); x[1] = bf16_hi(u.x); x[2] = bf16_lo(u.y); x[3] = bf16_hi(u.y);
            x[4] = bf16_lo(u.z); x[5] = bf16_hi(u.z); x[6] = bf16_lo(u.w); x[7] = bf16_hi(u.w);
        } else {
            x[0] = __uint_as_float(r.w[0].x); x[1] = __uint_as_float(r.w[0].y);
            x[2] = __uint_as_float(r.w[0].z); x[3] = __uint_as_float(r.w[0].w);
            x[4] = __uint_as_float(r.w[1].x); x[5] = __uint_as_float(r.w[1].y);
            x[6] = __uint_as_float(r.w[1].z); x[7] = __uint_as_float(r.w[1].w);
        }
#pragma unroll
        for (int i = 0; i < 8; ++i)
            if (base + i >= V) x[i] = -INFINITY;
    } else {
        mload8<BF16, VEC>(row, V, base, x);
    }
}

template <int LAYOUT>
__device__ __forceinline__ double clock_f64(uint32_t V, uint32_t slot, uint32_t v, uint32_t k0, uint32_t k1) {
    return LAYOUT == 0 ? tree_clock_f64(V, slot, v, k0, k1) : flat_clock_f64(slot, v, k0, k1);
}
template <int LAYOUT>
__device__ __forceinline__ float clock_f32(uint32_t V, uint32_t slot, uint32_t v, uint32_t k0, uint32_t k1) {
    return LAYOUT == 0 ? tree_clock_f32(V, slot, v, k0, k1) : flat_clock_f32(slot, v, k0, k1);
}

__device__ __forceinline__ bool lexless(double s, int v, int j, double s2, int v2, int j2) {
    return s < s2 || (s == s2 && (v < v2 || (v == v2 && j < j2)));
}

// (a list longer than kMCand is counted, not stored: the caller tightens theta and
// lists again)
__device__ __forceinline__ void push_cand(MShared& sm, int v, float x) {
    const int i = atomicAdd(&sm.n_cand, 1);
    if (i < kMCand) {
        sm.cand_v[i] = v;
        sm.cand_x[i] = x;
    }
}

// The candidates of one 8-token chunk (lane's part of a surviving group): chunk
// minimum (mc, pc), slot-0 token clocks, scores against theta.
template <int LAYOUT>
__device__ __forceinline__ void eval_chunk(MShared& sm, const MpfrArgs& a, const float (&x)[8], uint32_t chunk,
                                           float mg, uint32_t pg, float shift, uint32_t k0, uint32_t k1) {
    const uint32_t V = (uint32_t)a.V;
    const uint32_t cs = chunk * 8u, ce = node_end(kShift1, chunk, V);
    if (cs >= V) return;
    float cmax = -INFINITY;
    for (uint32_t t = 0; t < ce - cs; ++t) cmax = fmaxf(cmax, x[t]);
    if (cmax == -INFINITY) return;
    const float theta = sm.theta;
    float mc = 0.f;
    uint32_t pc = 0u;
    if constexpr (LAYOUT == 0) {
        child_min_f32(mg, pg, 1, chunk, cs, ce, 0u, k0, k1, mc, pc);
        if (ln_f32(mc) - (cmax - shift) * a.invT > theta) return;
    } else {
        if (kLnClockFloor - (cmax - shift) * a.invT > theta) return;
    }
#pragma unroll
    for (uint32_t h = 0; h < 2; ++h) {
        const Words w = LAYOUT == 0 ? philox(chunk, 0u, 8u + h, kDomainTree, k0, k1)
                                    : philox((cs >> 2) + h, 0u, 0u, kDomainFlat, k0, k1);
        const uint32_t ws[4] = {w.w0, w.w1, w.w2, w.w3};
#pragma unroll
        for (uint32_t t = 0; t < 4; ++t) {
            const uint32_t v = cs + 4u * h + t;
            const float xv = x[4 * h + t];
            if (v >= ce || xv == -INFINITY) continue;
            float E;
            if constexpr (LAYOUT == 0)
                E = v == pc ? mc : mc + exp1_f32(ws[t]);
            else
                E = exp1_f32(ws[t]);
            if (ln_f32(E) - (xv - shift) * a.invT <= theta) push_cand(sm, (int)v, xv);
        }
    }
}

// Stream one row: log-sum-exp at T (to *lse_out when non-null), the maximum of every
// 128-token group (to gm, in LDS or global memory) and the row maximum (returned to
// every thread).  red_* are LDS scratch of kMBlock / 64 entries.
template <bool BF16, bool VEC>
__device__ __forceinline__ float mstream_row(const unsigned char* row, int V, float invT, float* gm, float* lse_out,
                                             float* red_m, float* red_s, float* red_x, float* rowmax) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int ng = (V + 127) / 128;
    const float c2 = invT * 1.4426950408889634f;
    float mrun = -INFINITY, srun = 0.f, xmax = -INFINITY;
    const int nstep = (V + 2047) / 2048;
    // software-pipelined: the next four units' raw words are loaded before the current
    // four are reduced (words past the row are never used)
    MRaw<BF16, VEC> wn[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) mraw_load<BF16, VEC>(row, V, q * 2048 + 8 * tid, wn[q]);
    for (int st0 = 0; st0 < nstep; st0 += 4) {
        float x[4][8];
#pragma unroll
        for (int q = 0; q < 4; ++q) mraw_unpack<BF16, VEC>(row, V, (st0 + q) * 2048 + 8 * tid, wn[q], x[q]);
        if (st0 + 4 < nstep) {
#pragma unroll
            for (int q = 0; q < 4; ++q) mraw_load<BF16, VEC>(row, V, (st0 + 4 + q) * 2048 + 8 * tid, wn[q]);
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            if (st0 + q >= nstep) break;
            float um = x[q][0];
#pragma unroll
            for (int i = 1; i < 8; ++i) um = fmaxf(um, x[q][i]);
            const float g = row16_max(um);
            const int gi = (st0 + q) * 16 + (tid >> 4);
            if ((lane & 15) == 0 && gi < ng) gm[gi] = g;
            xmax = fmaxf(xmax, um);
            if (um > -INFINITY) {
                const float mn = fmaxf(mrun, um * c2);
                float acc = mrun == -INFINITY ? 0.f : srun * __builtin_amdgcn_exp2f(mrun - mn);
#pragma unroll
                for (int i = 0; i < 8; ++i) acc += __builtin_amdgcn_exp2f(fmaf(x[q][i], c2, -mn));
                srun = acc;
                mrun = mn;
            }
        }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        const float om = __shfl_xor(mrun, off), os = __shfl_xor(srun, off);
        xmax = fmaxf(xmax, __shfl_xor(xmax, off));
        const float mn = fmaxf(mrun, om);
        if (mn > -INFINITY) {
            srun = (mrun == -INFINITY ? 0.f : srun * __builtin_amdgcn_exp2f(mrun - mn)) +
                   (om == -INFINITY ? 0.f : os * __builtin_amdgcn_exp2f(om - mn));
            mrun = mn;
        }
    }
    if (lane == 0) {
        red_m[wave] = mrun;
        red_s[wave] = srun;
        red_x[wave] = xmax;
    }
    __syncthreads();
    if (tid == 0) {
        float m = red_m[0], sacc = red_s[0], xm = red_x[0];
        for (int w = 1; w < kMBlock / 64; ++w) {
            xm = fmaxf(xm, red_x[w]);
            const float om = red_m[w], os = red_s[w], mn = fmaxf(m, om);
            if (mn > -INFINITY) {
                sacc = (m == -INFINITY ? 0.f : sacc * __builtin_amdgcn_exp2f(m - mn)) +
                       (om == -INFINITY ? 0.f : os * __builtin_amdgcn_exp2f(om - mn));
                m = mn;
            }
        }
        *rowmax = xm;
        if (lse_out) *lse_out = m == -INFINITY ? -INFINITY : (m + __builtin_amdgcn_logf(sacc)) * 0.69314718055994531f;
    }
    __syncthreads();
    return *rowmax;
}

// Seed groups of a row: the largest group of each eighth of the row (lowest index on
// ties; -1 when the eighth has no finite logit), 32 lanes per eighth.  Every thread of
// the workgroup calls it; no barrier.
__device__ __forceinline__ void seed_groups(const float* gm, int ng, int* seed_g) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int r = 2 * wave + (lane >> 5), l32 = lane & 31;
    const int g0 = r * ng / kSeeds, g1 = (r + 1) * ng / kSeeds;
    float bv = -INFINITY;
    int bg = 0x7FFFFFFF;
    for (int g = g0 + l32; g < g1; g += 32)
        if (gm[g] > bv) {
            bv = gm[g];
            bg = g;
        }
#pragma unroll
    for (int off = 16; off > 0; off >>= 1) {
        const float ov = __shfl_xor(bv, off);
        const int og = __shfl_xor(bg, off);
        if (ov > bv || (ov == bv && og < bg)) {
            bv = ov;
            bg = og;
        }
    }
    if (l32 == 0) seed_g[r] = bv == -INFINITY ? -1 : bg;
}

// Each seed group's largest token (its lowest index holding the maximum), 16 lanes per
// group (after a barrier that published seed_g).  Every thread calls it.
template <bool BF16, bool VEC>
__device__ __forceinline__ void seed_tokens(const unsigned char* row, int V, const float* gm, const int* seed_g,
                                            int* seed_tok) {
    const int tid = threadIdx.x;
    if (tid < kSeeds * 16) {
        const int i = tid >> 4, sub = tid & 15, g = seed_g[i];
        int tk = 0x7FFFFFFF;
        if (g >= 0) {
            float x[8];
            const int base = g * 128 + sub * 8;
            mload8<BF16, VEC>(row, V, base, x);
#pragma unroll
            for (int t = 7; t >= 0; --t)
                if (base + t < V && x[t] == gm[g]) tk = base + t;
        }
#pragma unroll
        for (int off = 8; off > 0; off >>= 1) tk = min(tk, __shfl_xor(tk, off));
        if (sub == 0) seed_tok[i] = g >= 0 && tk != 0x7FFFFFFF ? tk : -1;
    }
}

// Values that may be read while their launch still runs (the streamed rows' maxima and
// seeds, the drafts of a launch that runs every depth) are tagged words: relaxed
// device-scope atomics are coherent across the XCDs without cache write-back, and
// the tag (the call's epoch) tells a reader that this call's value has landed.
__device__ __forceinline__ void mst_dev(uint64_t* p, uint64_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t mld_dev(const uint64_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t mld_dev_u32(const uint32_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The call's epoch for its tagged words: one more than the last recorded (1 .. 2^32-1).
__device__ __forceinline__ uint32_t next_epoch(const MpfrArgs& a) {
    const uint32_t last = mld_dev_u32(a.ctrl + kCtrlMpfrEpoch);
    return last == 0xFFFFFFFFu ? 1u : last + 1u;
}

// The last workgroup of a launch to leave resets the exit count and records the epoch.
__device__ __forceinline__ void record_epoch(const MpfrArgs& a, uint32_t ep) {
    const uint32_t old = __hip_atomic_fetch_add(a.ctrl + kCtrlMpfrExited, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (old == gridDim.x - 1) {
        __hip_atomic_store(a.ctrl + kCtrlMpfrExited, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(a.ctrl + kCtrlMpfrEpoch, ep, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

// The streaming launch of a call over the draft rows of depths [s_begin, s_begin +
// s_count), depth-major (the first depth's rows are handed out first), one row per
// workgroup or (stream_grid) several, writing each row's group maxima, maximum and
// seed tokens as tagged words and its LSE.  It never waits.
template <bool BF16, bool VEC>
__global__ __launch_bounds__(kMBlock) void mpfr_stream_kernel(MpfrArgs a) {
    __shared__ float red_m[kMBlock / 64], red_s[kMBlock / 64], red_x[kMBlock / 64], rowmax;
    __shared__ float gm[kMaxGroups];
    __shared__ int seed_g[kSeeds], seed_tok[kSeeds];
    __shared__ uint32_t ep_s;
    const int n = a.B * a.K;
    const int row_end = n * a.s_count;
    const int ng = (a.V + 127) / 128;
    const size_t esize = BF16 ? 2 : 4;
    if (threadIdx.x == 0) ep_s = next_epoch(a);
    // rows blockIdx.x, blockIdx.x + gridDim.x, ...: with fewer workgroups than rows, the
    // first depths' rows land first
    for (int r = (int)blockIdx.x; r < row_end; r += (int)gridDim.x) {
        const int s = a.s_begin + r / n, b = (r % n) / a.K, k = r % a.K;
        const unsigned char* row = (const unsigned char*)a.logits +
                                   (((size_t)b * a.K + k) * a.s_count + (size_t)(s - a.s_begin)) * (size_t)a.V * esize;
        const size_t rid = ((size_t)b * a.K + k) * a.gamma + s;
        const float xm = mstream_row<BF16, VEC>(row, a.V, a.invT, gm, a.draft_lse ? a.draft_lse + rid : nullptr,
                                                red_m, red_s, red_x, &rowmax);
        // (mstream_row ends with a barrier: the group maxima and the epoch are in LDS)
        const uint64_t tag = (uint64_t)ep_s << 32;
        for (int g = threadIdx.x; g < ng; g += kMBlock) mst_dev(a.row_gm + rid * ng + g, tag | __float_as_uint(gm[g]));
        if (threadIdx.x == 0) mst_dev(a.row_max + rid, tag | __float_as_uint(xm));
        // the row's seed tokens, for every context this row may serve
        seed_groups(gm, ng, seed_g);
        __syncthreads();
        seed_tokens<BF16, VEC>(row, a.V, gm, seed_g, seed_tok);
        __syncthreads();
        if (threadIdx.x < kSeeds)
            mst_dev(a.row_seed + rid * kSeeds + threadIdx.x, tag | (uint32_t)seed_tok[threadIdx.x]);
        __syncthreads();  // gm and the seeds are reused by the next row
    }
    if (a.stream_records_epoch && threadIdx.x == 0) record_epoch(a, ep_s);
}

// Bounded wait for the draft of row rid; on timeout the call's error bit 0 is set and
// the token reads as -1.
__device__ __forceinline__ int wait_draft(const MpfrArgs& a, size_t rid, uint32_t ep) {
    uint64_t v = mld_dev(a.tok_slot + rid);
    for (uint32_t i = 0; (uint32_t)(v >> 32) != ep; ++i) {
        if (i >= a.spin_limit) {
            __hip_atomic_fetch_or(a.ctrl + kCtrlCallErrors, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            return -1;
        }
        __builtin_amdgcn_s_sleep(2);
        v = mld_dev(a.tok_slot + rid);
    }
    return (int)(uint32_t)v;
}

// Payload of a word the streaming launch wrote.  A launch that runs every depth may
// run beside the streaming launch: it waits (bounded) for this call's tag.  Launches of
// one depth follow the streaming launch in stream order and read the payload.
__device__ __forceinline__ uint32_t row_word(const MpfrArgs& a, const uint64_t* p, uint32_t ep) {
    if (!a.tok_slot) return (uint32_t)*p;
    uint64_t v = mld_dev(p);
    for (uint32_t i = 0; (uint32_t)(v >> 32) != ep; ++i) {
        if (i >= a.spin_limit) {
            __hip_atomic_fetch_or(a.ctrl + kCtrlCallErrors, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            break;
        }
        __builtin_amdgcn_s_sleep(2);
        v = mld_dev(p);
    }
    return (uint32_t)v;
}

// Depth s of path k of sequence b (every thread of the workgroup calls it; its early
// returns are uniform).  ep: the launch's epoch when it runs every depth.
template <bool BF16, bool VEC, int LAYOUT>
__device__ __forceinline__ void mpfr_depth(const MpfrArgs& a, MShared& sm, float* gm, int b, int k, int s, uint32_t ep) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const uint32_t V = (uint32_t)a.V;
    const int ng = (a.V + 127) / 128, n3 = (ng + 15) / 16, n4 = (n3 + 15) / 16;
    const size_t esize = BF16 ? 2 : 4;
    const unsigned char* row = (const unsigned char*)a.logits +
                               (((size_t)b * a.K + k) * a.s_count + (size_t)(s - a.s_begin)) * (size_t)a.V * esize;

    // ---- the context of path k: the paths whose drafts at depths < s equal its own
    // (depths of this launch: from their tagged slots, when one launch runs every depth)
    for (int e = tid; e < a.K * s; e += kMBlock) {
        const size_t rid = ((size_t)b * a.K + e / s) * a.gamma + e % s;
        sm.path_tok[e] = a.tok_slot && e % s >= a.s_begin ? wait_draft(a, rid, ep) : a.draft_tokens[rid];
    }
    for (int e = tid; e < a.m; e += kMBlock) sm.pre[e] = a.prefix[(size_t)b * a.m + e];
    if (tid == 0) sm.n_l4 = sm.n_l3 = sm.n_cand = 0;
    __syncthreads();
    if (wave == 0) {
        bool same = lane < a.K;
        for (int d = 0; d < s && same; ++d) same = sm.path_tok[lane * s + d] == sm.path_tok[k * s + d];
        const uint64_t bal = __ballot(same);
        if (lane == 0) sm.mask = (uint32_t)bal;
    }

    if (a.row_gm) {
        // the row was streamed ahead (group maxima, maximum and LSE): only the context's
        // lowest path goes on, loading them
        __syncthreads();
        if (k != __ffs((int)sm.mask) - 1) return;  // uniform
        const size_t rid = ((size_t)b * a.K + k) * a.gamma + s;
        // four loads in flight per thread, then a wait only for words not yet tagged
        for (int g0 = tid; g0 < ng; g0 += 4 * kMBlock) {
            uint64_t w[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int g = g0 + i * kMBlock;
                w[i] = g < ng ? (a.tok_slot ? mld_dev(a.row_gm + rid * ng + g) : a.row_gm[rid * ng + g]) : 0;
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int g = g0 + i * kMBlock;
                if (g < ng) {
                    const uint32_t x = a.tok_slot && (uint32_t)(w[i] >> 32) != ep ? row_word(a, a.row_gm + rid * ng + g, ep)
                                                                                   : (uint32_t)w[i];
                    gm[g] = __uint_as_float(x);
                }
            }
        }
        if (tid == 0) sm.rowmax = __uint_as_float(row_word(a, a.row_max + rid, ep));
        if (tid < kSeeds) {
            const int tk = (int)row_word(a, a.row_seed + rid * kSeeds + tid, ep);
            sm.seed_tok[tid] = tk;
            sm.seed_g[tid] = tk >= 0 ? tk / 128 : -1;
        }
    } else {
        // ---- stream the row: log-sum-exp, group maxima, row maximum
        __syncthreads();
        mstream_row<BF16, VEC>(row, a.V, a.invT, gm,
                               a.draft_lse ? a.draft_lse + ((size_t)b * a.K + k) * a.gamma + s : nullptr, sm.red_m,
                               sm.red_s, sm.red_x, &sm.rowmax);
    }
    __syncthreads();
    const uint32_t mask = sm.mask;
    if (k != __ffs((int)mask) - 1) return;  // the context's lowest path samples it (uniform)
    const int nu = __popc(mask);
    const float shift = sm.rowmax;
    if (shift == -INFINITY) {  // no finite logit: every draft of the context is -1
        if (tid < nu) sm.samples[tid] = -1;
    } else {
        // ---- context key (key, t, last m tokens of prefix || path), level maxima, seeds
        if (tid == 0) {
            uint32_t k0 = (uint32_t)a.key, k1 = (uint32_t)(a.key >> 32);
            const uint64_t t = (uint64_t)(a.start_pos[b] + s);
            fold(k0, k1, (uint32_t)t, (uint32_t)(t >> 32), 0u);
            for (int i = 0; i < a.m; ++i) {
                const int g = s + i;  // index in prefix (m tokens) || path (s tokens)
                const int w = g < a.m ? sm.pre[g] : sm.path_tok[k * s + (g - a.m)];
                fold(k0, k1, (uint32_t)w, (uint32_t)i, 1u);
            }
            sm.kappa0 = k0;
            sm.kappa1 = k1;
        }
        for (int t = tid; t < n3; t += kMBlock) {
            float mx = -INFINITY;
            for (int g = 16 * t; g < min(ng, 16 * t + 16); ++g) mx = fmaxf(mx, gm[g]);
            sm.m3[t] = mx;
        }
        if (!a.row_seed) seed_groups(gm, ng, sm.seed_g);
        __syncthreads();
        for (int t = tid; t < n4; t += kMBlock) {
            float mx = -INFINITY;
            for (int i = 16 * t; i < min(n3, 16 * t + 16); ++i) mx = fmaxf(mx, sm.m3[i]);
            sm.m4[t] = mx;
        }
        if (!a.row_seed) seed_tokens<BF16, VEC>(row, a.V, gm, sm.seed_g, sm.seed_tok);
        __syncthreads();
        const uint32_t k0 = sm.kappa0, k1 = sm.kappa1;
        // seed arrivals in float32: E_j for every (seed, j < nu), the cumulative sums in
        // arrival order, then every score at once.  theta only has to bound the context's
        // nu-th smallest score from above: float32 scores are within the pruning margin
        // of the exact ones (the same assumption as every float32 bound of the race), and
        // theta carries one margin for that on top of its own.  A seed token holds its
        // group's maximum, so its logit is that maximum.
        for (int e = tid; e < kSeeds * nu; e += kMBlock) {
            const int i = e / nu, j = e % nu, v = sm.seed_tok[i];
            sm.pair[i * 32 + j] = v >= 0 ? (double)clock_f32<LAYOUT>(V, (uint32_t)j, (uint32_t)v, k0, k1) : 0.0;
        }
        __syncthreads();
        if (tid < kSeeds) {
            float G = 0.f;
            for (int j = 0; j < nu; ++j) {
                G += (float)sm.pair[tid * 32 + j];
                sm.pair[tid * 32 + j] = (double)G;
            }
        }
        __syncthreads();
        {
            const int i = tid >> 5, j = tid & 31, v = sm.seed_tok[i];
            static_assert(kSeeds * 32 == kMBlock, "one seed arrival slot per thread");
            sm.pair[tid] = v >= 0 && j < nu
                               ? (double)(ln_f32((float)sm.pair[tid]) - (gm[sm.seed_g[i]] - shift) * a.invT)
                               : INFINITY;
        }
        __syncthreads();
        if (wave == 0) {
            // theta = the nu-th smallest seed score (nu rounds of a wave minimum)
            double v4[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) v4[q] = sm.pair[lane + 64 * q];
            double th = INFINITY;
            for (int r = 0; r < nu; ++r) {
                double mv = v4[0];
                int mi = lane;
#pragma unroll
                for (int q = 1; q < 4; ++q)
                    if (v4[q] < mv) {
                        mv = v4[q];
                        mi = lane + 64 * q;
                    }
#pragma unroll
                for (int off = 32; off > 0; off >>= 1) {
                    const double ov = __shfl_xor(mv, off);
                    const int oi = __shfl_xor(mi, off);
                    if (ov < mv || (ov == mv && oi < mi)) {
                        mv = ov;
                        mi = oi;
                    }
                }
                th = mv;
                if ((mi & 63) == lane) v4[mi >> 6] = INFINITY;
            }
            if (lane == 0) sm.theta = th == INFINITY ? INFINITY : (float)th + 2.f * kMMargin;
        }
        __syncthreads();

        // ---- list every token whose slot-0 score can reach theta.  A list longer than
        // kMCand tightens theta to the nu-th smallest exact slot-0 score among its first
        // kMCand tokens (nu real arrivals, so still an upper bound) and lists again.
        float rm = 0.f;
        uint32_t rp = 0u;
        if constexpr (LAYOUT == 0) root_min_f32(V, 0u, k0, k1, rm, rp);
        for (int attempt = 0;; ++attempt) {
            if (tid == 0) sm.n_l4 = sm.n_l3 = sm.n_cand = 0;
            __syncthreads();
            if constexpr (LAYOUT == 0) {
                if (tid < n4) {
                    float m;
                    uint32_t p;
                    const uint32_t cs = (uint32_t)tid << kShift4;
                    child_min_f32(rm, rp, 4, (uint32_t)tid, cs, node_end(kShift4, (uint32_t)tid, V), 0u, k0, k1, m, p);
                    if (ln_f32(m) - (sm.m4[tid] - shift) * a.invT <= sm.theta)
                        sm.l4[atomicAdd(&sm.n_l4, 1)] = MNode{(uint32_t)tid, m, p};
                }
                __syncthreads();
                if (tid < sm.n_l4 * 16) {
                    const MNode pa = sm.l4[tid >> 4];
                    const uint32_t i3 = pa.i * 16u + (uint32_t)(tid & 15);
                    if ((int)i3 < n3) {
                        float m;
                        uint32_t p;
                        child_min_f32(pa.m, pa.p, 3, i3, i3 << kShift3, node_end(kShift3, i3, V), 0u, k0, k1, m, p);
                        if (ln_f32(m) - (sm.m3[i3] - shift) * a.invT <= sm.theta)
                            sm.l3[atomicAdd(&sm.n_l3, 1)] = MNode{i3, m, p};
                    }
                }
                __syncthreads();
                const int nl3 = sm.n_l3;
                for (int n0 = 0; n0 < nl3; n0 += 16) {  // 16 level-3 nodes (256 groups) per batch
                    if (tid == 0) sm.n_lg = 0;
                    __syncthreads();
                    const int e = n0 * 16 + tid;
                    if (e < nl3 * 16) {
                        const MNode pa = sm.l3[e >> 4];
                        const uint32_t g = pa.i * 16u + (uint32_t)(e & 15);
                        if ((int)g < ng && ln_f32(pa.m) - (gm[g] - shift) * a.invT <= sm.theta) {
                            float m;
                            uint32_t p;
                            child_min_f32(pa.m, pa.p, 2, g, g << kShift2, node_end(kShift2, g, V), 0u, k0, k1, m, p);
                            if (ln_f32(m) - (gm[g] - shift) * a.invT <= sm.theta)
                                sm.lg[atomicAdd(&sm.n_lg, 1)] = MNode{g, m, p};
                        }
                    }
                    __syncthreads();
                    const int nlg = sm.n_lg;
                    for (int g0 = 0; g0 < nlg; g0 += 16) {  // 16 lanes per group, one chunk each
                        const int gi = g0 + (tid >> 4);
                        if (gi < nlg) {
                            const MNode gn = sm.lg[gi];
                            const uint32_t chunk = gn.i * 16u + (uint32_t)(tid & 15);
                            float x[8];
                            mload8<BF16, VEC>(row, a.V, (int)(chunk * 8u), x);
                            eval_chunk<0>(sm, a, x, chunk, gn.m, gn.p, shift, k0, k1);
                        }
                    }
                    __syncthreads();
                }
            } else {
                for (int g0 = 0; g0 < ng; g0 += 16) {
                    const int g = g0 + (tid >> 4);
                    if (g < ng && kLnClockFloor - (gm[g] - shift) * a.invT <= sm.theta) {
                        const uint32_t chunk = (uint32_t)g * 16u + (uint32_t)(tid & 15);
                        float x[8];
                        mload8<BF16, VEC>(row, a.V, (int)(chunk * 8u), x);
                        eval_chunk<1>(sm, a, x, chunk, 0.f, 0u, shift, k0, k1);
                    }
                }
            }
            __syncthreads();
            if (sm.n_cand <= kMCand) break;
            if (attempt == 3) {  // still too many: the samples may be wrong, and the call says so
                if (tid == 0)
                    __hip_atomic_fetch_or(a.ctrl + kCtrlCallErrors, kMErrCand, __ATOMIC_RELAXED,
                                          __HIP_MEMORY_SCOPE_AGENT);
                break;
            }
            // tighter theta: exact slot-0 scores of the stored tokens, nu-th smallest
            for (int c = tid; c < kMCand; c += kMBlock)
                sm.cand_s[c] = log(clock_f64<LAYOUT>(V, 0u, (uint32_t)sm.cand_v[c], k0, k1)) -
                               ((double)sm.cand_x[c] - (double)shift) / (double)a.T;
            __syncthreads();
            double th = INFINITY;
            for (int r = 0; r < nu; ++r) {
                double bs = INFINITY;
                int bi = 0x7FFFFFFF;
                for (int c = tid; c < kMCand; c += kMBlock)
                    if (sm.cand_s[c] < bs) {
                        bs = sm.cand_s[c];
                        bi = c;
                    }
#pragma unroll
                for (int off = 32; off > 0; off >>= 1) {
                    const double os = __shfl_xor(bs, off);
                    const int oi = __shfl_xor(bi, off);
                    if (os < bs || (os == bs && oi < bi)) {
                        bs = os;
                        bi = oi;
                    }
                }
                if (lane == 0) {
                    sm.red_d[wave] = bs;
                    sm.red_i[wave] = bi;
                }
                __syncthreads();
                if (tid == 0) {
                    for (int w = 1; w < kMBlock / 64; ++w)
                        if (sm.red_d[w] < bs || (sm.red_d[w] == bs && sm.red_i[w] < bi)) {
                            bs = sm.red_d[w];
                            bi = sm.red_i[w];
                        }
                    if (bi >= 0 && bi < kMCand) sm.cand_s[bi] = INFINITY;
                    sm.red_d[0] = bs;
                }
                __syncthreads();
                th = sm.red_d[0];
                __syncthreads();
            }
            if (tid == 0) sm.theta = fminf(sm.theta, (float)th + kMMargin);
            __syncthreads();
        }

        // ---- exact arrivals of the listed tokens; nu rounds of the lexicographic minimum
        const int nc = min(sm.n_cand, kMCand);
        if (nc * nu <= kMBlock) {
            // every arrival j < nu of every listed token at once (one fp64 clock per
            // thread, in the seed array, free by now), the cumulative sums in arrival
            // order (the same sums as one arrival at a time), then the nu smallest
            // (score, token, arrival) by one wave: the same samples in the same order
            const int t = tid, c = t / nu, j = t % nu;
            if (t < nc * nu) sm.pair[t] = clock_f64<LAYOUT>(V, (uint32_t)j, (uint32_t)sm.cand_v[c], k0, k1);
            __syncthreads();
            if (t < nc) {
                double G = 0.0;
                for (int i = 0; i < nu; ++i) {
                    G += sm.pair[t * nu + i];
                    sm.pair[t * nu + i] = G;
                }
            }
            __syncthreads();
            if (t < nc * nu)
                sm.pair[t] = log(sm.pair[t]) - ((double)sm.cand_x[c] - (double)shift) / (double)a.T;
            __syncthreads();
            if (wave == 0) {
                double ps[4];
                int pv[4], pj[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int e = lane + 64 * q;
                    const bool ok = e < nc * nu;
                    ps[q] = ok ? sm.pair[e] : INFINITY;
                    pv[q] = ok ? sm.cand_v[e / nu] : 0x7FFFFFFF;
                    pj[q] = ok ? e % nu : 0x7FFFFFFF;
                }
                for (int r = 0; r < nu; ++r) {
                    double bs = INFINITY;
                    int bv = 0x7FFFFFFF, bj = 0x7FFFFFFF, bi = -1;
#pragma unroll
                    for (int q = 0; q < 4; ++q)
                        if (lexless(ps[q], pv[q], pj[q], bs, bv, bj)) {
                            bs = ps[q];
                            bv = pv[q];
                            bj = pj[q];
                            bi = lane + 64 * q;
                        }
#pragma unroll
                    for (int off = 32; off > 0; off >>= 1) {
                        const double os = __shfl_xor(bs, off);
                        const int ov = __shfl_xor(bv, off), oj = __shfl_xor(bj, off), oi = __shfl_xor(bi, off);
                        if (lexless(os, ov, oj, bs, bv, bj)) {
                            bs = os;
                            bv = ov;
                            bj = oj;
                            bi = oi;
                        }
                    }
                    if (lane == 0) sm.samples[r] = bs < INFINITY ? bv : -1;
                    if (bi >= 0 && (bi & 63) == lane) {
#pragma unroll
                        for (int q = 0; q < 4; ++q)
                            if (q == (bi >> 6)) ps[q] = INFINITY;
                    }
                }
            }
        } else {
        for (int c = tid; c < nc; c += kMBlock) {
            const int v = sm.cand_v[c];
            const double G = clock_f64<LAYOUT>(V, 0u, (uint32_t)v, k0, k1);
            sm.cand_g[c] = G;
            sm.cand_j[c] = 0;
            sm.cand_s[c] = log(G) - ((double)sm.cand_x[c] - (double)shift) / (double)a.T;
        }
        __syncthreads();
        for (int r = 0; r < nu; ++r) {
            double bs = INFINITY;
            int bv = 0x7FFFFFFF, bj = 0x7FFFFFFF, bi = -1;
            for (int c = tid; c < nc; c += kMBlock)
                if (lexless(sm.cand_s[c], sm.cand_v[c], sm.cand_j[c], bs, bv, bj)) {
                    bs = sm.cand_s[c];
                    bv = sm.cand_v[c];
                    bj = sm.cand_j[c];
                    bi = c;
                }
#pragma unroll
            for (int off = 32; off > 0; off >>= 1) {
                const double os = __shfl_xor(bs, off);
                const int ov = __shfl_xor(bv, off), oj = __shfl_xor(bj, off), oi = __shfl_xor(bi, off);
                if (lexless(os, ov, oj, bs, bv, bj)) {
                    bs = os;
                    bv = ov;
                    bj = oj;
                    bi = oi;
                }
            }
            if (lane == 0) {
                sm.red_d[wave] = bs;
                sm.red_v[wave] = bv;
                sm.red_j[wave] = bj;
                sm.red_i[wave] = bi;
            }
            __syncthreads();
            if (tid == 0) {
                for (int w = 1; w < kMBlock / 64; ++w)
                    if (lexless(sm.red_d[w], sm.red_v[w], sm.red_j[w], bs, bv, bj)) {
                        bs = sm.red_d[w];
                        bv = sm.red_v[w];
                        bj = sm.red_j[w];
                        bi = sm.red_i[w];
                    }
                sm.samples[r] = bs < INFINITY ? bv : -1;
                if (bi >= 0 && bs < INFINITY) {
                    // the winner's next arrival (or none past nu)
                    const int j = sm.cand_j[bi] + 1;
                    if (j < nu) {
                        const double G = sm.cand_g[bi] + clock_f64<LAYOUT>(V, (uint32_t)j, (uint32_t)bv, k0, k1);
                        sm.cand_g[bi] = G;
                        sm.cand_j[bi] = j;
                        sm.cand_s[bi] = log(G) - ((double)sm.cand_x[bi] - (double)shift) / (double)a.T;
                    } else {
                        sm.cand_s[bi] = INFINITY;
                    }
                }
            }
            __syncthreads();
        }
        }
    }
    __syncthreads();
    if (tid == 0) {
        // the context's r-th sample goes to its r-th path
        uint32_t mm = mask;
        for (int r = 0; r < nu; ++r) {
            const int kk = __ffs((int)mm) - 1;
            mm &= mm - 1u;
            const size_t rid = ((size_t)b * a.K + kk) * a.gamma + s;
            a.draft_tokens[rid] = sm.samples[r];
            if (a.tok_slot) mst_dev(a.tok_slot + rid, ((uint64_t)ep << 32) | (uint32_t)sm.samples[r]);
        }
    }
}

// One workgroup per (sequence, path).  Without tok_slot: depth a.s only.  With it:
// every depth of the call in turn, each depth's contexts formed from the drafts of the
// earlier depths as they land; waits are only for workgroups of the same launch, so
// the launcher uses this form only when all of them can be resident together.  The
// last workgroup to leave resets the exit count and records the launch's epoch.
template <bool BF16, bool VEC, int LAYOUT>
__global__ __launch_bounds__(kMBlock, 3) void mpfr_draft_kernel(MpfrArgs a) {
    __shared__ MShared sm;
    extern __shared__ __align__(16) float gm[];  // the row's group maxima (dynamic: one per group)
    const int b = (int)blockIdx.x / a.K, k = (int)blockIdx.x % a.K;
    if (!a.tok_slot) {
        mpfr_depth<BF16, VEC, LAYOUT>(a, sm, gm, b, k, a.s, 0u);
        return;
    }
    if (threadIdx.x == 0) sm.epoch = next_epoch(a);
    __syncthreads();
    const uint32_t ep = sm.epoch;
    for (int s = a.s_begin; s < a.s_begin + a.s_count; ++s) {
        mpfr_depth<BF16, VEC, LAYOUT>(a, sm, gm, b, k, s, ep);
        __syncthreads();
    }
    if (threadIdx.x == 0) record_epoch(a, ep);
}

// The call's error bits to the sticky word and the caller's status word (for calls
// that end without a fused race kernel, whose last workgroup does this).
__global__ void finish_status_kernel(uint32_t* ctrl, uint32_t* status) {
    const uint32_t bits = __hip_atomic_exchange(ctrl + kCtrlCallErrors, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (bits) __hip_atomic_fetch_or(ctrl + kCtrlErrors, bits, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (status) *status = bits;
}

}  // namespace

namespace {

// Dynamic LDS of a sampling launch: the row's group maxima.
size_t mpfr_draft_smem(const MpfrArgs& a) { return (size_t)(((a.V + 127) / 128 + 3) & ~3) * sizeof(float); }

template <bool BF16, bool VEC, int LAYOUT>
hipError_t mpfr_fit(const MpfrArgs& a, bool* fits) {
    *fits = false;
    if (!a.row_gm || a.s_count < 2) return hipSuccess;
    int per_cu = 0, dev = 0, cus = 0;
    hipError_t e;
    if ((e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, mpfr_draft_kernel<BF16, VEC, LAYOUT>, kMBlock,
                                                          mpfr_draft_smem(a))) != hipSuccess)
        return e;
    if ((e = hipGetDevice(&dev)) != hipSuccess) return e;
    if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess) return e;
    *fits = (long)per_cu * cus >= (long)a.B * a.K;
    return hipSuccess;
}

// tok_slot set (the caller checked mpfr_all_depths_fit): one launch for every depth;
// otherwise one launch per depth.
template <bool BF16, bool VEC, int LAYOUT>
hipError_t mpfr_depths(MpfrArgs a, hipStream_t stream) {
    auto fn = mpfr_draft_kernel<BF16, VEC, LAYOUT>;
    const dim3 grid((unsigned)(a.B * a.K)), block(kMBlock);
    const size_t smem = mpfr_draft_smem(a);
    hipError_t e;
    if (a.tok_slot) {
        hipLaunchKernelGGL(fn, grid, block, smem, stream, a);
        return hipGetLastError();
    }
    for (int s = a.s_begin; s < a.s_begin + a.s_count; ++s) {
        a.s = s;
        hipLaunchKernelGGL(fn, grid, block, smem, stream, a);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace

hipError_t mpfr_all_depths_fit(const MpfrArgs& a, bool bf16, bool vec, int layout, bool* fits) {
    if (bf16) {
        if (vec) return layout == 0 ? mpfr_fit<true, true, 0>(a, fits) : mpfr_fit<true, true, 1>(a, fits);
        return layout == 0 ? mpfr_fit<true, false, 0>(a, fits) : mpfr_fit<true, false, 1>(a, fits);
    }
    if (vec) return layout == 0 ? mpfr_fit<false, true, 0>(a, fits) : mpfr_fit<false, true, 1>(a, fits);
    return layout == 0 ? mpfr_fit<false, false, 0>(a, fits) : mpfr_fit<false, false, 1>(a, fits);
}

hipError_t launch_mpfr_depths(MpfrArgs a, bool bf16, bool vec, int layout, hipStream_t stream) {
    if (bf16) {
        if (vec) return layout == 0 ? mpfr_depths<true, true, 0>(a, stream) : mpfr_depths<true, true, 1>(a, stream);
        return layout == 0 ? mpfr_depths<true, false, 0>(a, stream) : mpfr_depths<true, false, 1>(a, stream);
    }
    if (vec) return layout == 0 ? mpfr_depths<false, true, 0>(a, stream) : mpfr_depths<false, true, 1>(a, stream);
    return layout == 0 ? mpfr_depths<false, false, 0>(a, stream) : mpfr_depths<false, false, 1>(a, stream);
}

hipError_t launch_mpfr_stream(const MpfrArgs& a, bool bf16, bool vec, hipStream_t stream) {
    const int rows = a.B * a.K * a.s_count;
    const dim3 grid((unsigned)(a.stream_grid > 0 && a.stream_grid < rows ? a.stream_grid : rows)), block(kMBlock);
    if (bf16) {
        if (vec) hipLaunchKernelGGL((mpfr_stream_kernel<true, true>), grid, block, 0, stream, a);
        else hipLaunchKernelGGL((mpfr_stream_kernel<true, false>), grid, block, 0, stream, a);
    } else {
        if (vec) hipLaunchKernelGGL((mpfr_stream_kernel<false, true>), grid, block, 0, stream, a);
        else hipLaunchKernelGGL((mpfr_stream_kernel<false, false>), grid, block, 0, stream, a);
    }
    return hipGetLastError();
}

hipError_t launch_finish_status(uint32_t* ctrl, uint32_t* status, hipStream_t stream) {
    hipLaunchKernelGGL(finish_status_kernel, dim3(1), dim3(1), 0, stream, ctrl, status);
    return hipGetLastError();
}

}  // namespace psd
