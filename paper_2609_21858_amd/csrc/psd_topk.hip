// psd_topk.hip -- logit processing before the race: top-k, then top-p (gfx950).
//
// The paper's experiments race the processed distributions (temperature, top-k,
// top-p; Alg. "Batched-target direct-top-k MPFR speculative sampling"): every
// token outside a row's kept set has probability 0.  With at most 256 kept tokens
// per row the race needs no pruning, so this path has two kernels:
//  * topk_select_kernel, one workgroup per row, one pass over the row in HBM that
//    keeps only the maximum of every 128-token group; the top_k-th largest group
//    maximum bounds the row's top_k-th largest logit from below, so only the groups
//    whose maximum reaches it are read again and their logits that reach it are the
//    candidates (wave buffers in LDS: ballot and lane prefix, no atomics).  Block-wide
//    bisections over the candidates' keys and then their indices pick the k largest
//    (order-preserving keys, ties to the lowest index).  Rows whose ties at the cut
//    overflow the buffers are selected by exact radix passes instead.  Then the kept
//    list is sorted by (logit descending, index ascending), its top-p prefix and the
//    log-sum-exp of the kept set at the row's temperature are formed in fp64;
//  * the races over the lists, exact fp64 clocks of every (token, slot) -- distinct
//    drafters race slot k / all K slots, identical drafters draw each context's nu
//    samples from the cumulative clocks and race the targets on slot 0 -- then the
//    walk.  Distinct drafters (drafting, or with the shared target chain):
//    topk_chain_kernel, one workgroup per (sequence, chain) -- a draft path, or the
//    target chain, whose races four waves share while a fifth folds the next key --
//    then topk_walk_kernel (the walk, one wave per sequence, and the status word).
//    Identical drafters or per-path target rows: topk_race_kernel, one workgroup per
//    sequence with one wave per chain, depth by depth (identical drafters group the
//    paths into contexts at every depth).
#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>

#include "psd_device.hpp"
#include "psd_launch.hpp"
#include "psd_layout.hpp"

namespace psd {

namespace {

constexpr int kTBlock = 256;
constexpr int kUnroll = 4;  // 16-byte loads in flight per thread
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------- keys

// Order-preserving keys (larger value, larger key); -0 takes the key of +0, as the two
// compare equal.
__device__ __forceinline__ uint32_t key_f32(uint32_t u) {
    if (u == 0x80000000u) u = 0u;
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float val_f32(uint32_t k) {
    return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}
__device__ __forceinline__ float tload(const unsigned char* row, bool bf16, int v) {
    return bf16 ? __uint_as_float((uint32_t)((const uint16_t*)row)[v] << 16) : ((const float*)row)[v];
}

constexpr int kWaves = kTBlock / 64;
constexpr int kWaveCap = 512;  // candidates a wave holds

// ---------------------------------------------------------------- block helpers

constexpr int kMaxGroups = (1 << 19) / kGroupTokens;  // 128-token groups of the largest row
constexpr int kCandGroups = 2 * kMaxTopK;             // groups re-read for candidates

struct SelShared {
    union {
        struct {
            uint32_t key[kWaves][kWaveCap];  // each wave's candidates: order-preserving key,
            int32_t idx[kWaves][kWaveCap];   // token index
        } wb;
        int hist[2048];         // radix passes (the candidates are given up first)
        float gm[kMaxGroups];   // group maxima of the streaming pass
    } u;
    int tok[kMaxTopK];
    float val[kMaxTopK];
    union {
        struct {
            int stok[kMaxTopK];
            float sval[kMaxTopK];
        };
        int cgl[kCandGroups];  // groups holding candidates (before the kept list is sorted)
    };
    int red[2][kWaves];
    double dred[kWaves];
    double dsel;
    int s4[kWaves];
    int wcount[kWaves], wover[kWaves];
    int n_keep, n_fin;
    uint32_t tsel;  // a key threshold found by one wave
    uint32_t prefix;
    int above;
};

__device__ __forceinline__ int wave_incl(int x) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(x, o);
        if (lane >= o) x += y;
    }
    return x;
}

// Lanes below this one whose bit is set in m.
__device__ __forceinline__ int lanes_below(uint64_t m) {
    return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// Entries of the wave (Q per lane) passing a test, counted with ballots (scalar
// popcounts: no lane shuffles).
template <int Q, typename F>
__device__ __forceinline__ int wave_count(F&& pass) {
    int c = 0;
#pragma unroll
    for (int q = 0; q < Q; ++q) c += __popcll(__ballot(pass(q)));
    return c;
}

// Sum over the workgroup of a wave-uniform count; the two LDS buffers alternate
// (parity `it`), so one barrier per call suffices.
__device__ __forceinline__ int block_sum_waves(SelShared& sm, int wave_total, int& it) {
    int* r = sm.red[it & 1];
    ++it;
    if ((threadIdx.x & 63) == 0) r[threadIdx.x >> 6] = wave_total;
    __syncthreads();
    int t = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) t += r[w];
    return t;
}

// Inclusive prefix sum of one int per thread (thread order); *total gets the sum.
__device__ __forceinline__ int block_incl_sum(SelShared& sm, int x, int& total) {
    const int wave = threadIdx.x >> 6;
    x = wave_incl(x);
    if ((threadIdx.x & 63) == 63) sm.s4[wave] = x;
    __syncthreads();
    int base = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
        if (w < wave) base += sm.s4[w];
        tot += sm.s4[w];
    }
    __syncthreads();
    total = tot;
    return x + base;
}

// Inclusive prefix sum of one double per thread (thread order); *total gets the sum.
__device__ __forceinline__ double block_incl_sum_f64(SelShared& sm, double x, double& total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const double y = __shfl_up(x, o);
        if (lane >= o) x += y;
    }
    if (lane == 63) sm.dred[wave] = x;
    __syncthreads();
    double base = 0.0, tot = 0.0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
        if (w < wave) base += sm.dred[w];
        tot += sm.dred[w];
    }
    __syncthreads();
    total = tot;
    return x + base;
}

// ---------------------------------------------------------------- one-wave selection

// The need-th largest key class t of Q keys per lane (0: no entry) with the wave's
// ballots alone (no barrier): largest t (bits below kLow clear) with #{key >= t} >= need.
template <int Q, int kLow>
__device__ __forceinline__ uint32_t wave_kth_class(const uint32_t (&kk)[Q], int need) {
    uint32_t t = 0u;
    for (int bit = 31; bit >= kLow; --bit) {
        const uint32_t cand = t | (1u << bit);
        if (wave_count<Q>([&](int q) { return kk[q] >= cand; }) >= need) t = cand;
    }
    return t;
}

// ---------------------------------------------------------------- one-pass selection

// Keys of bf16 logits differ only in their top 16 bits (the low half is 0x0000 or
// 0xFFFF by sign), so searches over them stop at bit 16; one key class is one value.
template <bool BF16>
struct KeyBits {
    static constexpr int kLow = BF16 ? 16 : 0;
};

template <bool BF16>
__device__ __forceinline__ uint32_t elem_bits(const uint32_t (&w)[4], int i) {
    return BF16 ? ((i & 1) ? (w[i >> 1] & 0xFFFF0000u) : (w[i >> 1] << 16)) : w[i];
}

// Group maxima of the row (128-token groups) into sm.u.gm: one wave per 64 x EPT-token
// chunk in turn (wave w takes chunks w, w + 4, ...; four 16-byte loads per lane in
// flight), the maximum of each lane's tokens, then of the lanes of a group.  Only a
// maximum per token: the pass costs little more than reading the row.
template <bool BF16>
__device__ __forceinline__ void stream_group_max(SelShared& sm, const unsigned char* row, int V) {
    constexpr int EPT = BF16 ? 8 : 4, WCH = 64 * EPT, STEP = kWaves * kUnroll, LPG = kGroupTokens / EPT;
    constexpr size_t ES = BF16 ? 2 : 4;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const bool vec = ((uintptr_t)row & 15u) == 0;
    const int nch = (V + WCH - 1) / WCH, ng = (V + kGroupTokens - 1) / kGroupTokens;
    for (int c0 = w; c0 < nch; c0 += STEP) {
        uint32_t wv[kUnroll][4];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int base = (c0 + u * kWaves) * WCH + lane * EPT;
            if (vec && base + EPT <= V) {
                const u32x4 q = __builtin_nontemporal_load((const u32x4*)(row + (size_t)base * ES));
                wv[u][0] = q.x;
                wv[u][1] = q.y;
                wv[u][2] = q.z;
                wv[u][3] = q.w;
            } else {
#pragma unroll
                for (int i = 0; i < 4; ++i) wv[u][i] = BF16 ? 0xFF80FF80u : 0xFF800000u;  // -inf
#pragma unroll
                for (int i = 0; i < EPT; ++i) {
                    const int v = base + i;
                    if (v < V) {
                        if (BF16) {
                            const uint32_t h = ((const uint16_t*)row)[v];
                            wv[u][i >> 1] = (wv[u][i >> 1] & ~(0xFFFFu << (16 * (i & 1)))) | (h << (16 * (i & 1)));
                        } else {
                            wv[u][i] = ((const uint32_t*)row)[v];
                        }
                    }
                }
            }
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            float mx = __uint_as_float(elem_bits<BF16>(wv[u], 0));
#pragma unroll
            for (int i = 1; i < EPT; ++i) mx = fmaxf(mx, __uint_as_float(elem_bits<BF16>(wv[u], i)));
            mx = row16_max(mx);
            if (LPG == 32) mx = fmaxf(mx, __shfl_xor(mx, 16));
            const int g = (c0 + u * kWaves) * (WCH / kGroupTokens) + lane / LPG;
            if (lane % LPG == 0 && g < ng) sm.u.gm[g] = mx;
        }
    }
}

// The candidates of the row's top-k set, without a per-logit pass over the row: t =
// the top_k-th largest key class among the group maxima (a bisection with ballot
// counts, in one wave when it holds every group maximum, else block-wide), so
// at least top_k logits reach t and every logit of the top-k set (ties at the cut
// included) reaches it too; only groups whose maximum reaches t can hold such a
// logit, and they are read again.  With fewer groups than top_k, every group with a
// finite logit is read again.  Their finite logits that reach t go to the wave
// buffers (ballot and lane prefix), as the per-logit selection would leave them.
// Returns false when the groups or the candidates do not fit (heavy ties at the
// cut); the caller then selects by radix passes.
template <bool BF16>
__device__ __forceinline__ bool select_candidates(SelShared& sm, const unsigned char* row, int V, int top_k) {
    constexpr int EPT = BF16 ? 8 : 4, LPG = kGroupTokens / EPT, GPW = 64 / LPG;  // groups per wave step
    constexpr int QG = kMaxGroups / kTBlock;
    constexpr size_t ES = BF16 ? 2 : 4;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int ng = (V + kGroupTokens - 1) / kGroupTokens;
    stream_group_max<BF16>(sm, row, V);
    __syncthreads();
    uint32_t kg[QG];
    bool fin[QG];
#pragma unroll
    for (int q = 0; q < QG; ++q) {
        const int g = tid + kTBlock * q;
        const float m = g < ng ? sm.u.gm[g] : -INFINITY;
        fin[q] = m >= -3.40282347e38f;  // a finite (or +inf) logit in the group; not NaN
        kg[q] = fin[q] ? key_f32(__float_as_uint(m)) : 0u;
    }
    int it = 0;
    uint32_t t = 0u;
    constexpr int QW = 16;  // group maxima per lane when one wave holds them all
    if (ng >= top_k && ng <= 64 * QW) {
        // one wave finds t over all the group maxima; the others wait at one barrier
        if (w == 0) {
            uint32_t kw[QW];
#pragma unroll
            for (int q = 0; q < QW; ++q) {
                const int g = lane + 64 * q;
                const float m = g < ng ? sm.u.gm[g] : -INFINITY;
                kw[q] = m >= -3.40282347e38f ? key_f32(__float_as_uint(m)) : 0u;
            }
            const uint32_t tw = wave_kth_class<QW, KeyBits<BF16>::kLow>(kw, top_k);
            if (lane == 0) sm.tsel = tw;
        }
        __syncthreads();
        t = sm.tsel;
    } else if (ng >= top_k) {
        for (int bit = 31; bit >= KeyBits<BF16>::kLow; --bit) {
            const uint32_t cand = t | (1u << bit);
            if (block_sum_waves(sm, wave_count<QG>([&](int q) { return fin[q] && kg[q] >= cand; }), it) >= top_k)
                t = cand;
        }
    }
    // the groups to read again, compacted (thread order)
    int nc = 0;
#pragma unroll
    for (int q = 0; q < QG; ++q) nc += fin[q] && kg[q] >= t;
    int n_cg;
    int off = block_incl_sum(sm, nc, n_cg) - nc;
    if (n_cg > kCandGroups) {
        if (tid == 0) sm.wover[0] = 1;
        __syncthreads();
        return false;
    }
#pragma unroll
    for (int q = 0; q < QG; ++q)
        if (fin[q] && kg[q] >= t) sm.cgl[off++] = tid + kTBlock * q;
    __syncthreads();  // (the group maxima are dead: the wave buffers reuse their space)
    // wave w reads groups w*GPW .. of every step of kWaves*GPW list entries
    uint32_t* bk = sm.u.wb.key[w];
    int32_t* bi = sm.u.wb.idx[w];
    const bool vec = ((uintptr_t)row & 15u) == 0;
    int cnt = 0;
    bool over = false;
    for (int e0 = w * GPW; e0 < n_cg; e0 += kWaves * GPW * kUnroll) {
        uint32_t wv[kUnroll][4];
        int base[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int e = e0 + u * kWaves * GPW + lane / LPG;
            base[u] = -1;
#pragma unroll
            for (int i = 0; i < 4; ++i) wv[u][i] = BF16 ? 0xFF80FF80u : 0xFF800000u;  // -inf
            if (e < n_cg && e < e0 + u * kWaves * GPW + GPW) {
                base[u] = sm.cgl[e] * kGroupTokens + (lane % LPG) * EPT;
                if (vec && base[u] + EPT <= V) {
                    const uint4 q = *(const uint4*)(row + (size_t)base[u] * ES);
                    wv[u][0] = q.x;
                    wv[u][1] = q.y;
                    wv[u][2] = q.z;
                    wv[u][3] = q.w;
                } else {
#pragma unroll
                    for (int i = 0; i < EPT; ++i) {
                        const int v = base[u] + i;
                        if (v < V) {
                            if (BF16) {
                                const uint32_t h = ((const uint16_t*)row)[v];
                                wv[u][i >> 1] = (wv[u][i >> 1] & ~(0xFFFFu << (16 * (i & 1)))) | (h << (16 * (i & 1)));
                            } else {
                                wv[u][i] = ((const uint32_t*)row)[v];
                            }
                        }
                    }
                }
            }
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
#pragma unroll
            for (int i = 0; i < EPT; ++i) {
                const uint32_t bits = elem_bits<BF16>(wv[u], i);
                const float x = __uint_as_float(bits);
                const bool pass = base[u] >= 0 && x >= -3.40282347e38f && key_f32(bits) >= t && !over;
                const uint64_t m = __ballot(pass);
                if (m) {
                    if (pass) {
                        const int pos = cnt + lanes_below(m);
                        bk[pos] = key_f32(bits);
                        bi[pos] = base[u] + i;
                    }
                    cnt += __popcll(m);
                }
                if (cnt > kWaveCap - 64) {  // ties at the cut: give up (radix passes)
                    over = true;
                    cnt = 0;
                }
            }
        }
    }
    if (lane == 0) {
        sm.wcount[w] = cnt;
        sm.wover[w] = over ? 1 : 0;
    }
    __syncthreads();
    bool ok = true;
#pragma unroll
    for (int q = 0; q < kWaves; ++q) ok = ok && !sm.wover[q];
    return ok;
}

// Exact radix selection of the need = min(top_k, finite logits) largest (ties to the
// lowest index) into sm.tok / sm.val, unsorted: three digit passes (11, 11, 10 bits)
// find the need-th largest key, a fourth collects.  Reads the row four times.
// Returns need.
template <bool BF16>
__device__ int radix_select(SelShared& sm, const unsigned char* row, int V, int top_k) {
    const int tid = threadIdx.x;
    const int shifts[3] = {21, 10, 0};
    const int widths[3] = {11, 11, 10};
    if (tid == 0) {
        sm.prefix = 0u;
        sm.above = 0;
        sm.n_fin = 0;
    }
    int need = 0;
    for (int pass = 0; pass < 3; ++pass) {
        const int nb = 1 << widths[pass];
        for (int i = tid; i < nb; i += kTBlock) sm.u.hist[i] = 0;
        __syncthreads();
        const uint32_t pre = sm.prefix;
        const int hi_shift = shifts[pass] + widths[pass];  // bits above this digit must equal the prefix
        int nf = 0;
        for (int v = tid; v < V; v += kTBlock) {
            const float x = tload(row, BF16, v);
            if (x == -INFINITY) continue;
            ++nf;
            const uint32_t k = key_f32(__float_as_uint(x));
            if (hi_shift < 32 && (k >> hi_shift) != (pre >> hi_shift)) continue;
            atomicAdd(&sm.u.hist[(k >> shifts[pass]) & (uint32_t)(nb - 1)], 1);
        }
        if (pass == 0) atomicAdd(&sm.n_fin, nf);
        __syncthreads();
        if (pass == 0) need = min(top_k, sm.n_fin);
        if (need == 0) return 0;
        if (tid == 0) {
            int acc = sm.above, b = nb - 1;
            for (; b > 0; --b) {
                if (acc + sm.u.hist[b] >= need) break;
                acc += sm.u.hist[b];
            }
            sm.above = acc;
            sm.prefix = pre | ((uint32_t)b << shifts[pass]);
        }
        __syncthreads();
    }
    const uint32_t thr = sm.prefix;
    const int n_eq_take = need - sm.above;
    if (tid == 0) sm.n_keep = 0;
    __syncthreads();
    int ties_before = 0;
    for (int c0 = 0; c0 < V; c0 += kTBlock * 8) {
        float x[8];
        int nt = 0;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int v = c0 + tid * 8 + i;
            x[i] = v < V ? tload(row, BF16, v) : -INFINITY;
            nt += x[i] != -INFINITY && key_f32(__float_as_uint(x[i])) == thr;
        }
        int total;
        const int incl = block_incl_sum(sm, nt, total);
        int rank = ties_before + incl - nt;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            if (x[i] == -INFINITY) continue;
            const uint32_t k = key_f32(__float_as_uint(x[i]));
            bool keep = k > thr;
            if (k == thr) keep = rank++ < n_eq_take;
            if (keep) {
                const int j = atomicAdd(&sm.n_keep, 1);
                if (j < kMaxTopK) {
                    sm.tok[j] = c0 + tid * 8 + i;
                    sm.val[j] = x[i] == 0.0f ? 0.0f : x[i];
                }
            }
        }
        ties_before += total;
    }
    __syncthreads();
    return need;
}

// One row: kept list, its length and the LSE of the kept set.
template <bool BF16>
__global__ __launch_bounds__(kTBlock) void topk_select_kernel(TopkSelectArgs a) {
    __shared__ SelShared sm;
    const int tid = threadIdx.x;
    const bool s1 = (int)blockIdx.x >= a.seg[0].n_rows;
    const TopkSegment& G = s1 ? a.seg[1] : a.seg[0];
    const int r = (int)blockIdx.x - (s1 ? a.seg[0].n_rows : 0);
    const unsigned char* row = (const unsigned char*)G.logits + (size_t)r * a.V * (BF16 ? 2 : 4);
    const int rid = G.row_id_base + (G.group > 0 ? (r / G.group) * G.group_stride + r % G.group : r);
    const int lse_at = G.lse_index_base + (G.group > 0 ? (r / G.group) * G.lse_group_stride + r % G.group : r);

    int it = 0;
    int need;
    if (!select_candidates<BF16>(sm, row, a.V, a.top_k)) {
        __syncthreads();  // the candidate buffers are reused by the radix passes
        if (tid == 0 && a.radix_rows) atomicAdd(a.radix_rows, 1u);
        need = radix_select<BF16>(sm, row, a.V, a.top_k);
    } else {
        // the union of the wave buffers holds every logit at least the row's top_k-th
        // largest (ties included), or every finite logit when there are fewer
        constexpr int Q = kWaves * kWaveCap / kTBlock;
        constexpr int PW = kWaveCap / kTBlock;  // entries of one wave's buffer per thread
        uint32_t kk[Q];
        int32_t ii[Q];
        int tot = 0;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) tot += sm.wcount[w];
        need = min(a.top_k, tot);
        constexpr int QW = 4;  // candidates per lane when one wave holds them all
        if (need > 0 && tot <= 64 * QW) {
            // one wave: the same bisections over the concatenated buffers, with ballots
            if (tid < 64) {
                const int lane = tid;
                const int c0 = sm.wcount[0], c1 = c0 + sm.wcount[1], c2 = c1 + sm.wcount[2];
                uint32_t kk[QW];
                int32_t ii[QW];
#pragma unroll
                for (int q = 0; q < QW; ++q) {
                    const int j = lane + 64 * q;
                    const int bw = j < c0 ? 0 : j < c1 ? 1 : j < c2 ? 2 : 3;
                    const int p = j - (bw == 0 ? 0 : bw == 1 ? c0 : bw == 2 ? c1 : c2);
                    const bool ok = j < tot;
                    kk[q] = ok ? sm.u.wb.key[bw][p] : 0u;
                    ii[q] = ok ? sm.u.wb.idx[bw][p] : 0;
                }
                const uint32_t t = wave_kth_class<QW, KeyBits<BF16>::kLow>(kk, need);
                const uint32_t t_up = t + (1u << KeyBits<BF16>::kLow);
                const int n_gt = wave_count<QW>([&](int q) { return kk[q] >= t_up; });
                const int n_ge = wave_count<QW>([&](int q) { return kk[q] >= t; });
                const int take = need - n_gt;
                int xmax = 0x7FFFFFFF;
                if (n_ge - n_gt > take) {
                    int x = 0;
                    for (int bit = 18; bit >= 0; --bit) {
                        const int cand = x | (1 << bit);
                        if (wave_count<QW>([&](int q) { return kk[q] >= t && kk[q] < t_up && ii[q] < cand; }) < take)
                            x = cand;
                    }
                    xmax = x;
                }
                int off = 0;
#pragma unroll
                for (int q = 0; q < QW; ++q) {
                    const bool keep = kk[q] >= t_up || (kk[q] >= t && ii[q] <= xmax);
                    const uint64_t m = __ballot(keep);
                    const int pos = off + lanes_below(m);
                    if (keep && pos < kMaxTopK) {
                        sm.tok[pos] = ii[q];
                        sm.val[pos] = val_f32(kk[q]);
                    }
                    off += __popcll(m);
                }
            }
            __syncthreads();
        } else {
#pragma unroll
            for (int q = 0; q < Q; ++q) {
                const int w = q / PW, p = tid + kTBlock * (q % PW);
                const bool ok = p < sm.wcount[w];
                kk[q] = ok ? sm.u.wb.key[w][p] : 0u;
                ii[q] = ok ? sm.u.wb.idx[w][p] : 0;
            }
            if (need > 0) {
                // the need-th largest key class: largest t with #{key >= t} >= need
                uint32_t t = 0u;
                for (int bit = 31; bit >= KeyBits<BF16>::kLow; --bit) {
                    const uint32_t cand = t | (1u << bit);
                    if (block_sum_waves(sm, wave_count<Q>([&](int q) { return kk[q] >= cand; }), it) >= need) t = cand;
                }
                // keys of the next class up (key >= t_up) are strictly larger logits
                const uint32_t t_up = t + (1u << KeyBits<BF16>::kLow);
                const int n_gt = block_sum_waves(sm, wave_count<Q>([&](int q) { return kk[q] >= t_up; }), it);
                const int n_ge = block_sum_waves(sm, wave_count<Q>([&](int q) { return kk[q] >= t; }), it);
                const int take = need - n_gt;  // ties at t to keep, lowest indices first
                int xmax = 0x7FFFFFFF;         // keep the ties with index <= xmax
                if (n_ge - n_gt > take) {
                    // the take-th smallest index among the tied entries: largest x with #{index < x} < take
                    int x = 0;
                    for (int bit = 18; bit >= 0; --bit) {
                        const int cand = x | (1 << bit);
                        if (block_sum_waves(sm, wave_count<Q>([&](int q) {
                                                return kk[q] >= t && kk[q] < t_up && ii[q] < cand;
                                            }),
                                            it) < take)
                            x = cand;
                    }
                    xmax = x;
                }
                int kc = 0;
#pragma unroll
                for (int q = 0; q < Q; ++q) kc += kk[q] >= t_up || (kk[q] >= t && ii[q] <= xmax);
                int total;
                int off = block_incl_sum(sm, kc, total) - kc;
#pragma unroll
                for (int q = 0; q < Q; ++q)
                    if ((kk[q] >= t_up || (kk[q] >= t && ii[q] <= xmax)) && off < kMaxTopK) {
                        sm.tok[off] = ii[q];
                        sm.val[off] = val_f32(kk[q]);
                        ++off;
                    }
                __syncthreads();
            }
        }
    }
    if (need == 0) {
        if (tid == 0) {
            a.list_len[rid] = 0;
            a.list_lse[rid] = -INFINITY;
            if (G.lse_out) G.lse_out[lse_at] = -INFINITY;
        }
        return;
    }
    const int n = need;  // both branches leave exactly need entries
    // sort by (logit descending, index ascending): each entry's rank by counting
    if (tid < n) {
        const float xv = sm.val[tid];
        const int tv = sm.tok[tid];
        int rk = 0;
        for (int j = 0; j < n; ++j) rk += sm.val[j] > xv || (sm.val[j] == xv && sm.tok[j] < tv);
        sm.stok[rk] = tv;
        sm.sval[rk] = xv;
    }
    __syncthreads();
    // top-p on the sorted list: the shortest prefix whose normalised mass at T reaches
    // top_p; then the LSE of the kept set (fp64)
    const double T = (double)G.T;
    const double z0 = (double)sm.sval[0] / T;
    const double e = tid < n ? exp((double)sm.sval[tid] / T - z0) : 0.0;
    double tot;
    const double inc = block_incl_sum_f64(sm, e, tot);
    int keep = n;
    if (a.top_p < 1.0f)
        keep = min(n, block_sum_waves(sm, __popcll(__ballot(tid < n && inc / tot < (double)a.top_p)), it) + 1);
    if (tid == keep - 1) sm.dsel = inc;
    __syncthreads();
    if (tid == 0) {
        const float lse = (float)(z0 + log(sm.dsel));
        a.list_len[rid] = keep;
        a.list_lse[rid] = lse;
        if (G.lse_out) G.lse_out[lse_at] = lse;
    }
    int32_t* out_tok = a.list_tok + (size_t)rid * a.cap;
    float* out_val = a.list_val + (size_t)rid * a.cap;
    if (tid < keep) {
        out_tok[tid] = sm.stok[tid];
        out_val[tid] = sm.sval[tid];
    }
}

// ---------------------------------------------------------------- races over the lists

template <int LAYOUT>
__device__ __forceinline__ double tclock(uint32_t V, uint32_t slot, uint32_t v, uint32_t k0, uint32_t k1) {
    return LAYOUT == 0 ? tree_clock_f64(V, slot, v, k0, k1) : flat_clock_f64(slot, v, k0, k1);
}

__device__ __forceinline__ bool tlex(double s, int v, int j, double s2, int v2, int j2) {
    return s < s2 || (s == s2 && (v < v2 || (v == v2 && j < j2)));
}

// Lexicographic minimum of (s, v, j) over the wave, with its entry c; every lane
// returns the same result (a strict total order on distinct (v, j)).
__device__ __forceinline__ void wave_lexmin(double& s, int& v, int& j, int& c) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        const double os = __shfl_xor(s, o);
        const int ov = __shfl_xor(v, o), oj = __shfl_xor(j, o), oc = __shfl_xor(c, o);
        if (tlex(os, ov, oj, s, v, j)) {
            s = os;
            v = ov;
            j = oj;
            c = oc;
        }
    }
}

struct RaceShared {
    int path[32 * 33];    // drafts of each path ([path][depth])
    int chain[33];        // shared target chain
    int pchain[32 * 33];  // per-path target chains
    double ts[8];         // partial minima of a shared-chain target race, one per target wave
    int tv[8], tj[8];
    int pre[16];          // the sequence's context window before the block (m <= 16)
    uint32_t tp[2][2];    // the shared chain's next key without its newest token (by depth parity)
};

// Context key of the token at absolute position t whose previous tokens are the last
// m of prefix (m tokens, copied to LDS in pre) || path[0 .. d), folded up to window
// position n (n = m: the whole key; n = m - 1: all but the newest token); every lane
// of the wave computes it.
__device__ __forceinline__ void list_key(const TopkRaceArgs& a, const int* pre, int64_t t, const int* path, int d,
                                         uint32_t& k0, uint32_t& k1, int n) {
    k0 = (uint32_t)a.key;
    k1 = (uint32_t)(a.key >> 32);
    fold(k0, k1, (uint32_t)(uint64_t)t, (uint32_t)((uint64_t)t >> 32), 0u);
    for (int i = 0; i < n; ++i) {
        const int g = d + i;  // index in prefix || path
        const int w = g < a.m ? pre[g] : path[g - a.m];
        fold(k0, k1, (uint32_t)w, (uint32_t)i, 1u);
    }
}

// The race of one row's list over slots [slot0, slot0 + nslots) -- argmin of
// ln E_j[v] - l_v / T (exact, fp64) -- over the (token, slot) entries of 64-entry units
// part, part + nparts, ... by one wave.  Returns the wave's winning token (-1 when it
// has none) and, when asked, its score and slot.
template <int LAYOUT>
__device__ int wave_race(const TopkRaceArgs& a, int rid, int slot0, int nslots, float T, uint32_t k0, uint32_t k1,
                         int part = 0, int nparts = 1, double* out_s = nullptr, int* out_j = nullptr) {
    const int lane = threadIdx.x & 63;
    const int n = a.list_len[rid];
    const int* lt = a.list_tok + (size_t)rid * a.cap;
    const float* lv = a.list_val + (size_t)rid * a.cap;
    double bs = INFINITY;
    int bv = 0x7FFFFFFF, bj = 0x7FFFFFFF, bc = -1;
    for (int e = part * 64 + lane; e < n * nslots; e += 64 * nparts) {
        const int c = e / nslots, j = slot0 + e % nslots;
        const int v = lt[c];
        const double s = log(tclock<LAYOUT>((uint32_t)a.V, (uint32_t)j, (uint32_t)v, k0, k1)) - (double)lv[c] / (double)T;
        if (tlex(s, v, j, bs, bv, bj)) {
            bs = s;
            bv = v;
            bj = j;
            bc = c;
        }
    }
    wave_lexmin(bs, bv, bj, bc);
    if (out_s) {
        *out_s = bs;
        *out_j = bj;
    }
    return bs < INFINITY ? bv : -1;
}

// A lane's first (token, slot) entry of a list race, loaded ahead: the list's length
// and the token and logit of the lane's entry (its index clamped into the row's list,
// so the loads never wait for the length and never leave the list).
struct ListHead {
    int n, v;
    float x;
};

__device__ __forceinline__ ListHead list_head(const TopkRaceArgs& a, int rid, int nslots, int part) {
    const int c = min((part * 64 + (int)(threadIdx.x & 63)) / nslots, a.cap - 1);
    return ListHead{a.list_len[rid], a.list_tok[(size_t)rid * a.cap + c], a.list_val[(size_t)rid * a.cap + c]};
}

// wave_race with the lane's first entry taken from h (loaded while the previous race
// of the chain ran); later entries are loaded in place.
template <int LAYOUT>
__device__ int wave_race_h(const TopkRaceArgs& a, const ListHead& h, int rid, int slot0, int nslots, float T,
                           uint32_t k0, uint32_t k1, int part, int nparts, double* out_s, int* out_j) {
    const int lane = threadIdx.x & 63;
    const int n = h.n;
    const int* lt = a.list_tok + (size_t)rid * a.cap;
    const float* lv = a.list_val + (size_t)rid * a.cap;
    // (token, slot) packed as token * 32 + slot (tokens < 2^19, slots < 32): the same
    // order, one word less in each shuffle step
    double bs = INFINITY;
    int bvj = 0x7FFFFFFF;
    for (int e = part * 64 + lane, first = 1; e < n * nslots; e += 64 * nparts, first = 0) {
        const int c = e / nslots, j = slot0 + e % nslots;
        const int v = first ? h.v : lt[c];
        const float x = first ? h.x : lv[c];
        const double s = log(tclock<LAYOUT>((uint32_t)a.V, (uint32_t)j, (uint32_t)v, k0, k1)) - (double)x / (double)T;
        const int vj = (v << 5) | j;
        if (s < bs || (s == bs && vj < bvj)) {
            bs = s;
            bvj = vj;
        }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        const double os = __shfl_xor(bs, o);
        const int ovj = __shfl_xor(bvj, o);
        if (os < bs || (os == bs && ovj < bvj)) {
            bs = os;
            bvj = ovj;
        }
    }
    *out_s = bs;
    *out_j = bs < INFINITY ? (bvj & 31) : 0x7FFFFFFF;
    return bs < INFINITY ? (bvj >> 5) : -1;
}

// The nu MPFR samples of one context from its row's list, by one wave: the nu
// smallest of ln G_{v,j} - l_v / T over (v, j < nu), G_{v,j} = E_0[v] + ... + E_j[v];
// the r-th goes to the r-th path of `members` (ascending) at depth s.
template <int LAYOUT>
__device__ void wave_mpfr(const TopkRaceArgs& a, RaceShared& sm, int rid, uint32_t members, int s, float T,
                          uint32_t k0, uint32_t k1) {
    constexpr int Q = kMaxTopK / 64;
    const int lane = threadIdx.x & 63;
    const int n = a.list_len[rid];
    const int nu = __popc(members);
    const int* lt = a.list_tok + (size_t)rid * a.cap;
    const float* lv = a.list_val + (size_t)rid * a.cap;
    double Gs[Q], sc[Q], lT[Q];
    int tok[Q], jj[Q];
#pragma unroll
    for (int q = 0; q < Q; ++q) {
        const int c = lane + 64 * q;
        jj[q] = 0;
        if (c < n) {
            tok[q] = lt[c];
            lT[q] = (double)lv[c] / (double)T;
            Gs[q] = tclock<LAYOUT>((uint32_t)a.V, 0u, (uint32_t)tok[q], k0, k1);
            sc[q] = log(Gs[q]) - lT[q];
        } else {
            tok[q] = 0x7FFFFFFF;
            lT[q] = 0.0;
            Gs[q] = 0.0;
            sc[q] = INFINITY;
        }
    }
    uint32_t mm = members;
    for (int r = 0; r < nu; ++r) {
        double bs = INFINITY;
        int bv = 0x7FFFFFFF, bj = 0x7FFFFFFF, bc = -1;
#pragma unroll
        for (int q = 0; q < Q; ++q)
            if (tlex(sc[q], tok[q], jj[q], bs, bv, bj)) {
                bs = sc[q];
                bv = tok[q];
                bj = jj[q];
                bc = lane + 64 * q;
            }
        wave_lexmin(bs, bv, bj, bc);
        const int member = __ffs((int)mm) - 1;
        mm &= mm - 1u;
        if (lane == 0) sm.path[member * 33 + s] = bs < INFINITY ? bv : -1;
        if (bs < INFINITY && lane == (bc & 63)) {
            // the winner's next arrival (one clock, then back into its register slot)
            const int qb = bc >> 6;
            int j = 0;
            double g = 0.0, l = 0.0;
#pragma unroll
            for (int q = 0; q < Q; ++q)
                if (q == qb) {
                    j = jj[q] + 1;
                    g = Gs[q];
                    l = lT[q];
                }
            double ns = INFINITY;
            if (j < nu) {
                g += tclock<LAYOUT>((uint32_t)a.V, (uint32_t)j, (uint32_t)bv, k0, k1);
                ns = log(g) - l;
            }
#pragma unroll
            for (int q = 0; q < Q; ++q)
                if (q == qb) {
                    Gs[q] = g;
                    sc[q] = ns;
                    jj[q] = j;
                }
        }
    }
}

template <int LAYOUT>
__global__ __launch_bounds__(512) void topk_race_kernel(TopkRaceArgs a) {
    __shared__ RaceShared sm;
    const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, w = tid >> 6, nw = (int)(blockDim.x >> 6);
    const int K = a.K, G = a.gamma;
    const int D = a.B * K * G;
    const int64_t t0 = a.start_pos[b];
    // drafts known before the call (depths < s_begin, or all of them as input)
    for (int e = tid; e < K * G; e += blockDim.x)
        sm.path[(e / G) * 33 + e % G] = a.draft_tokens[((size_t)b * K + e / G) * G + e % G];
    for (int e = tid; e < a.m; e += blockDim.x) sm.pre[e] = a.prefix[(size_t)b * a.m + e];
    __syncthreads();
    const bool per = a.target_rows > 1;
    const int tslots = a.mpfr ? 1 : K;
    // waves [dw, nw) share each shared-chain target race; the others race the drafts
    const int twv = a.target_rows == 1 ? a.target_waves : 0, dw = nw - twv;
    const int d_end = a.s_begin + a.s_count;
    const int s_lo = a.target_rows > 0 ? 0 : a.s_begin;
    const int s_hi = a.target_rows > 0 ? G : d_end - 1;
    uint32_t k0, k1;
    for (int s = s_lo; s <= s_hi; ++s) {
        if (s >= a.s_begin && s < d_end && w < dw) {
            for (int k = w; k < K; k += dw) {
                if (!a.mpfr) {
                    list_key(a, sm.pre, t0 + s, &sm.path[k * 33], s, k0, k1, a.m);
                    const int y = wave_race<LAYOUT>(a, (b * K + k) * G + s, k, 1, a.T_draft, k0, k1);
                    if (lane == 0) sm.path[k * 33 + s] = y;
                } else {
                    // the context of path k: the paths with its drafts at depths < s; its
                    // lowest path draws the context's samples (wave-uniform)
                    uint32_t members = 0u;
                    bool rep = true;
                    for (int q = 0; q < K; ++q) {
                        bool same = true;
                        for (int d = 0; d < s && same; ++d) same = sm.path[q * 33 + d] == sm.path[k * 33 + d];
                        if (same) {
                            members |= 1u << q;
                            if (q < k) rep = false;
                        }
                    }
                    if (!rep) continue;
                    list_key(a, sm.pre, t0 + s, &sm.path[k * 33], s, k0, k1, a.m);
                    wave_mpfr<LAYOUT>(a, sm, (b * K + k) * G + s, members, s, a.T_draft, k0, k1);
                }
            }
        }
        if (a.target_rows == 1 && w >= dw) {
            const int ti = w - dw;
            if (s > 0 && a.m > 0) {
                // the rest of the key was folded during the previous depth; its newest
                // token is the previous depth's target
                k0 = sm.tp[s & 1][0];
                k1 = sm.tp[s & 1][1];
                fold(k0, k1, (uint32_t)sm.chain[s - 1], (uint32_t)(a.m - 1), 1u);
            } else {
                list_key(a, sm.pre, t0 + s, sm.chain, s, k0, k1, a.m);
            }
            double ps;
            int pj;
            const int pv = wave_race<LAYOUT>(a, D + b * (G + 1) + s, 0, tslots, a.T_target, k0, k1, ti, twv, &ps, &pj);
            if (lane == 0) {
                sm.ts[ti] = ps;
                sm.tv[ti] = pv;
                sm.tj[ti] = pj;
            }
        }
        if (a.target_rows == 1 && w == 0 && a.m > 0 && s < G) {
            // the next depth's shared-chain key up to its newest token (this depth's
            // target, not known yet): folded here by a draft wave, which finishes its
            // races before the target waves do
            uint32_t p0, p1;
            list_key(a, sm.pre, t0 + s + 1, sm.chain, s + 1, p0, p1, a.m - 1);
            if (lane == 0) {  // (the other parity: this depth's key was read from it)
                sm.tp[(s + 1) & 1][0] = p0;
                sm.tp[(s + 1) & 1][1] = p1;
            }
        }
        if (per)
            for (int k = w; k < K; k += nw) {
                list_key(a, sm.pre, t0 + s, &sm.path[k * 33], s, k0, k1, a.m);
                const int y = wave_race<LAYOUT>(a, D + (b * K + k) * (G + 1) + s, 0, tslots, a.T_target, k0, k1);
                if (lane == 0) sm.pchain[k * 33 + s] = y;
            }
        __syncthreads();
        if (twv > 0) {
            // the shared-chain target of depth s: the lexicographic minimum of the waves' parts
            if (tid == 0) {
                double bs = sm.ts[0];
                int bv = sm.tv[0], bj = sm.tj[0];
                for (int i = 1; i < twv; ++i)
                    if (tlex(sm.ts[i], sm.tv[i], sm.tj[i], bs, bv, bj)) {
                        bs = sm.ts[i];
                        bv = sm.tv[i];
                        bj = sm.tj[i];
                    }
                sm.chain[s] = bs < INFINITY ? bv : -1;
            }
            __syncthreads();
        }
    }
    if (a.s_count > 0)
        for (int e = tid; e < K * a.s_count; e += blockDim.x) {
            const int k = e / a.s_count, s = a.s_begin + e % a.s_count;
            a.draft_tokens[((size_t)b * K + k) * G + s] = sm.path[k * 33 + s];
        }
    if (a.target_rows == 0 || tid != 0) return;
    auto target = [&](int k, int s) { return per ? sm.pchain[k * 33 + s] : sm.chain[s]; };
    if (a.target_tokens)
        for (int k = 0; k < (per ? K : 1); ++k)
            for (int s = 0; s <= G; ++s) a.target_tokens[((size_t)b * (per ? K : 1) + k) * (G + 1) + s] = target(k, s);
    // ---- the walk (as in the fused kernel)
    uint32_t act = K >= 32 ? 0xFFFFFFFFu : ((1u << K) - 1u);
    int tau = 0;
    bool done = false;
    for (int s = 0; s < G && !done; ++s) {
        const int y = target(__ffs((int)act) - 1, s);
        a.out_tokens[(size_t)b * (G + 1) + s] = y;
        tau = s + 1;
        if (y < 0) {
            done = true;
            break;
        }
        uint32_t na = 0u;
        for (int k = 0; k < K; ++k)
            if (((act >> k) & 1u) && sm.path[k * 33 + s] == y) na |= 1u << k;
        if (!na) {
            done = true;
            break;
        }
        act = na;
    }
    if (!done) {
        a.out_tokens[(size_t)b * (G + 1) + G] = target(__ffs((int)act) - 1, G);
        tau = G + 1;
    }
    for (int s = tau; s <= G; ++s) a.out_tokens[(size_t)b * (G + 1) + s] = -1;
    a.out_len[b] = tau;
}

// Distinct drafters, drafting only or with the shared target chain: one workgroup per
// (sequence, chain) -- a draft path (one wave) or the target chain (four waves sharing
// each race, a fifth folding the next key) -- so a sequence's chains run on different
// CUs rather than sharing one CU's SIMDs.  The chains of a sequence are independent
// (the target chain is keyed by its own prefix), so no workgroup waits for another;
// the walk runs in the next launch.
struct ChainShared {
    int path[33];          // this workgroup's chain: drafts of one path, or the targets
    int pre[16];           // the sequence's context window before the block (m <= 16)
    double ts[4];          // partial minima of a target race, one per wave
    int tv[4], tj[4];
    uint32_t tp[2][2];     // the chain's next key without its newest token (by depth parity)
};

constexpr int kChainWaves = 4;  // waves sharing each target race; one more folds the next key

template <int LAYOUT>
__global__ __launch_bounds__(64 * (kChainWaves + 1)) void topk_chain_kernel(TopkRaceArgs a) {
    __shared__ ChainShared sm;
    const int K = a.K, G = a.gamma;
    const int nd = a.s_count > 0 ? K : 0, R = nd + (a.target_rows == 1 ? 1 : 0);
    const int b = (int)blockIdx.x / R, r = (int)blockIdx.x % R;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int64_t t0 = a.start_pos[b];
    const int d_end = a.s_begin + a.s_count;
    for (int e = tid; e < a.m; e += blockDim.x) sm.pre[e] = a.prefix[(size_t)b * a.m + e];
    if (r < nd)
        for (int e = tid; e < a.s_begin; e += blockDim.x) sm.path[e] = a.draft_tokens[((size_t)b * K + r) * G + e];
    __syncthreads();
    uint32_t k0, k1;
    if (r < nd) {
        // draft path k: its races in depth order, by one wave (every lane keeps the
        // same copy of the path, so no lane reads another lane's LDS write)
        if (w != 0) return;
        const int k = r;
        ListHead h = list_head(a, (b * K + k) * G + a.s_begin, 1, 0);
        for (int s = a.s_begin; s < d_end; ++s) {
            list_key(a, sm.pre, t0 + s, sm.path, s, k0, k1, a.m);
            const ListHead hs = h;
            if (s + 1 < d_end) h = list_head(a, (b * K + k) * G + s + 1, 1, 0);  // the next depth's, in flight
            double ps;
            int pj;
            sm.path[s] = wave_race_h<LAYOUT>(a, hs, (b * K + k) * G + s, k, 1, a.T_draft, k0, k1, 0, 1, &ps, &pj);
        }
        for (int s = a.s_begin + lane; s < d_end; s += 64) a.draft_tokens[((size_t)b * K + k) * G + s] = sm.path[s];
        return;
    }
    // the shared target chain: each race's (token, slot) entries shared by the waves
    const int tslots = K;
    const int trow = a.B * K * G + b * (G + 1);
    ListHead h = list_head(a, trow, tslots, w);
    for (int s = 0; s <= G; ++s) {
        if (w == kChainWaves) {
            // the next depth's key up to its newest token (this race's winner), folded
            // while the other waves race
            if (a.m > 0 && s < G) {
                uint32_t p0, p1;
                list_key(a, sm.pre, t0 + s + 1, sm.path, s + 1, p0, p1, a.m - 1);
                if (lane == 0) {  // (the other parity: this depth's key was read from it)
                    sm.tp[(s + 1) & 1][0] = p0;
                    sm.tp[(s + 1) & 1][1] = p1;
                }
            }
            __syncthreads();
            __syncthreads();
            continue;
        }
        if (s > 0 && a.m > 0) {
            k0 = sm.tp[s & 1][0];
            k1 = sm.tp[s & 1][1];
            fold(k0, k1, (uint32_t)sm.path[s - 1], (uint32_t)(a.m - 1), 1u);
        } else {
            list_key(a, sm.pre, t0 + s, sm.path, s, k0, k1, a.m);
        }
        const ListHead hs = h;
        if (s < G) h = list_head(a, trow + s + 1, tslots, w);  // the next depth's, in flight
        double ps;
        int pj;
        const int pv = wave_race_h<LAYOUT>(a, hs, trow + s, 0, tslots, a.T_target, k0, k1, w, kChainWaves, &ps, &pj);
        if (lane == 0) {
            sm.ts[w] = ps;
            sm.tv[w] = pv;
            sm.tj[w] = pj;
        }
        __syncthreads();
        if (tid == 0) {
            double bs = sm.ts[0];
            int bv = sm.tv[0], bj = sm.tj[0];
            for (int i = 1; i < kChainWaves; ++i)
                if (tlex(sm.ts[i], sm.tv[i], sm.tj[i], bs, bv, bj)) {
                    bs = sm.ts[i];
                    bv = sm.tv[i];
                    bj = sm.tj[i];
                }
            sm.path[s] = bs < INFINITY ? bv : -1;
        }
        __syncthreads();
    }
    for (int s = tid; s <= G; s += blockDim.x) {
        a.chain[(size_t)b * (G + 1) + s] = sm.path[s];
        if (a.target_tokens) a.target_tokens[(size_t)b * (G + 1) + s] = sm.path[s];
    }
}

// The walk of every sequence over its drafts and shared-chain targets, then the call's
// error bits to the sticky word and the caller's status word.  One wave per sequence:
// its lanes load the sequence's targets and drafts into LDS together (one memory
// latency instead of one per depth), and lane 0 walks, as the fused kernel does.
constexpr int kWalkWaves = 4;
constexpr int kWalkVals = kMaxDepth + 32 * (kMaxDepth - 1);  // gamma + 1 targets, K <= 32 paths of gamma drafts

__global__ __launch_bounds__(64 * kWalkWaves) void topk_walk_kernel(TopkRaceArgs a) {
    __shared__ int32_t vals[kWalkWaves][kWalkVals];
    const int lane = (int)threadIdx.x & 63, wave = (int)threadIdx.x >> 6;
    const int b = (int)blockIdx.x * kWalkWaves + wave;
    const int K = a.K, G = a.gamma;
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        const uint32_t bits = __hip_atomic_exchange(a.ctrl + kCtrlCallErrors, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (bits) __hip_atomic_fetch_or(a.ctrl + kCtrlErrors, bits, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (a.status) *a.status = bits | (a.status_in ? *a.status_in : 0u);
    }
    const bool valid = b < a.B;
    int32_t* v = vals[wave];
    const int nt = G + 1, n = nt + K * G;  // n <= kWalkVals (K and gamma are checked by the caller)
    if (valid) {
        const int32_t* y = a.chain + (size_t)b * nt;
        const int32_t* d = a.draft_tokens + (size_t)b * K * G;
        for (int e = lane; e < n; e += 64) v[e] = e < nt ? y[e] : d[e - nt];
    }
    __syncthreads();
    if (!valid || lane != 0) return;
    const int32_t* d = v + nt;
    uint32_t act = K >= 32 ? 0xFFFFFFFFu : ((1u << K) - 1u);
    int tau = 0;
    bool done = false;
    for (int s = 0; s < G && !done; ++s) {
        const int ys = v[s];
        a.out_tokens[(size_t)b * (G + 1) + s] = ys;
        tau = s + 1;
        if (ys < 0) {
            done = true;
            break;
        }
        uint32_t na = 0u;
        for (int k = 0; k < K; ++k)
            if (((act >> k) & 1u) && d[k * G + s] == ys) na |= 1u << k;
        if (!na) {
            done = true;
            break;
        }
        act = na;
    }
    if (!done) {
        a.out_tokens[(size_t)b * (G + 1) + G] = v[G];
        tau = G + 1;
    }
    for (int s = tau; s <= G; ++s) a.out_tokens[(size_t)b * (G + 1) + s] = -1;
    a.out_len[b] = tau;
}

}  // namespace

hipError_t launch_walk(const TopkRaceArgs& a, hipStream_t stream) {
    hipLaunchKernelGGL(topk_walk_kernel, dim3((unsigned)((a.B + kWalkWaves - 1) / kWalkWaves)), dim3(64 * kWalkWaves), 0, stream, a);
    return hipGetLastError();
}

hipError_t launch_topk_select(const TopkSelectArgs& a, bool bf16, hipStream_t stream) {
    const int n = a.seg[0].n_rows + a.seg[1].n_rows;
    if (n <= 0) return hipSuccess;
    if (bf16)
        hipLaunchKernelGGL(topk_select_kernel<true>, dim3(n), dim3(kTBlock), 0, stream, a);
    else
        hipLaunchKernelGGL(topk_select_kernel<false>, dim3(n), dim3(kTBlock), 0, stream, a);
    return hipGetLastError();
}

hipError_t launch_topk_race(const TopkRaceArgs& a, int layout, hipStream_t stream) {
    hipError_t e;
    if (!a.mpfr && a.target_rows <= 1) {
        // one workgroup per (sequence, chain), then the walk and the status
        const int R = (a.s_count > 0 ? a.K : 0) + (a.target_rows == 1 ? 1 : 0);
        if (R > 0) {
            const dim3 grid((unsigned)(a.B * R)), block(64 * (kChainWaves + 1));
            if (layout == 0)
                hipLaunchKernelGGL(topk_chain_kernel<0>, grid, block, 0, stream, a);
            else
                hipLaunchKernelGGL(topk_chain_kernel<1>, grid, block, 0, stream, a);
            if ((e = hipGetLastError()) != hipSuccess) return e;
        }
        if (a.target_rows == 1) {
            hipLaunchKernelGGL(topk_walk_kernel, dim3((unsigned)((a.B + kWalkWaves - 1) / kWalkWaves)), dim3(64 * kWalkWaves), 0, stream, a);
            return hipGetLastError();
        }
        return launch_finish_status(a.ctrl, a.status, stream);
    }
    // identical drafters (contexts group paths at every depth) or per-path target rows:
    // one workgroup per sequence, at most 8 waves (the TREE clocks need more than 128
    // registers per lane): one per draft path, and for a shared target chain up to four
    // sharing each of its races (its K-slot races are the longest of a depth)
    TopkRaceArgs b = a;
    int waves;
    if (a.target_rows == 1) {
        b.target_waves = a.K >= 7 ? 1 : (8 - a.K < 4 ? 8 - a.K : 4);
        waves = (a.K < 8 - b.target_waves ? a.K : 8 - b.target_waves) + b.target_waves;
    } else {
        b.target_waves = 0;
        waves = a.K < 8 ? a.K : 8;
    }
    if (layout == 0)
        hipLaunchKernelGGL(topk_race_kernel<0>, dim3(a.B), dim3(64 * waves), 0, stream, b);
    else
        hipLaunchKernelGGL(topk_race_kernel<1>, dim3(a.B), dim3(64 * waves), 0, stream, b);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return launch_finish_status(a.ctrl, a.status, stream);
}

}  // namespace psd
