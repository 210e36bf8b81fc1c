// psd_race.hip -- fused draft + verify kernel of the keyed Poisson race (gfx950).
//
// One persistent kernel per call.  Workgroups pull work items from a global
// ticket counter; an item is one 32 KiB segment of one logits row.  Items are
// ordered depth-major (all rows of depth 0, then depth 1, ...), and the segments
// of a row are consecutive, so every row a race depends on holds lower tickets.
//
// Per segment (key-independent, HBM-streaming): coalesced 16-byte loads, the
// online log-sum-exp partial (max, sum of exp2) and the maximum logit of every
// 128-token group.  The workgroup that completes a row's last segment becomes the
// row's finisher: it merges the LSE partials, waits for the token its context
// needs (the previous depth of the same path or chain), folds the context key and
// runs the keyed race over the row's group maxima:
//
//  * TREE clocks: best-first by level.  A node's lower bound is
//    ln(min clock of the node) - max logit / T; only nodes whose bound can still
//    beat the best score found so far are expanded, and only the 128-token groups
//    that survive are re-read from memory (a few per row).
//  * FLAT clocks: every group whose bound ln(clock floor) - max logit / T can win
//    is re-read and its surviving tokens draw their Philox word.
//
// Pruning and candidate scores run in float32 with a safety margin; every
// candidate within the margin of the best is re-scored in float64 (clock rebuilt
// exactly, logit / T in double) and the winner is the lexicographic minimum of
// (score, token, slot) -- exact ties go to the lowest token, then slot.
//
// Paper passages: race = eq. EFR (Thm. "PFR reduces to EFR"); draft k races
// slot k and the target races all K slots (Prop. "heterogeneous PML bound",
// augmented space V x [K]); target chain keyed by its own prefix (stopping-time
// drafter invariance); walk = Alg. "Multi-Draft ... (Formal)".
#include <hip/hip_runtime.h>

#include <math.h>

#include "psd_device.hpp"
#include "psd_launch.hpp"
#include "psd_layout.hpp"

namespace psd {

namespace {

constexpr int kL4Cap = 512;   // <= 32 slots x 16 level-4 nodes
constexpr int kL3Cap = 512;
constexpr int kL2Cap = 256;
constexpr int kCandCap = 256;
constexpr float kMargin = 1e-3f;           // float32 pruning / candidate margin (score units)
constexpr uint32_t kSpinLimit = 1u << 22;  // bounded dependency wait
constexpr uint32_t kErrSpin = 1u, kErrCand = 2u;

struct Node {
    uint32_t id;  // (slot << 20) | node index
    float m;      // float32 minimum clock of the node
    uint32_t p;   // token holding that minimum
};

struct Shared {
    float m3[256];
    float m4[16];
    Node l4[kL4Cap];
    Node l3[kL3Cap];
    Node l2[kL2Cap];
    int cand_v[kCandCap];
    int cand_j[kCandCap];
    float cand_s[kCandCap];
    float root_m[32];
    uint32_t root_p[32];
    int32_t window[16];
    double red_s[kBlock / 64];
    int red_v[kBlock / 64];
    int red_j[kBlock / 64];
    float red_a[kBlock / 64];
    float red_b[kBlock / 64];
    int n_l4, n_l3, n_l2, n_cand;
    int best_key;
    int item, fin, last;
    int win_token, win_slot;
    int gstar;
    float rowmax;
    uint32_t kappa0, kappa1;
};

struct Row {
    int kind;  // 0 draft, 1 target
    int b, k, s;
    int row_id;
    const unsigned char* ptr;
    int slot0, nslots;
    float invT;
    float T;
};

__device__ __forceinline__ uint32_t* ctrl_of(const RaceArgs& a) { return (uint32_t*)(a.ws + a.L.ctrl); }

__device__ __forceinline__ void set_error(const RaceArgs& a, uint32_t bit) { atomicOr(ctrl_of(a) + 2, bit); }

// Cross-workgroup words (group maxima, LSE partials, tokens, flags, counters) are
// only touched with relaxed device-scope atomics, which are coherent across the
// XCDs without L2-wide write-back / invalidate.  Ordering between a producer's
// data and its flag comes from waiting for its stores to complete (s_waitcnt)
// before the flag is written; compiler fences keep the accesses in program order.
template <typename T>
__device__ __forceinline__ void st_dev(T* p, T v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
template <typename T>
__device__ __forceinline__ T ld_dev(const T* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void drain_memory() {
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_waitcnt(0);
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

__device__ __forceinline__ int target_row_id(const RaceArgs& a, int b, int k, int s) {
    const int D = a.B * a.K * a.gamma;
    return a.target_rows == 1 ? D + b * (a.gamma + 1) + s : D + (b * a.K + k) * (a.gamma + 1) + s;
}

__device__ __forceinline__ int draft_row_id(const RaceArgs& a, int b, int k, int s) {
    return (b * a.K + k) * a.gamma + s;
}

// Bounded wait until *flag != 0 (acquire).  On timeout an error bit is recorded
// and the caller proceeds, so every wave always terminates.
__device__ void wait_nonzero(const RaceArgs& a, const uint32_t* flag) {
    for (uint32_t i = 0;; ++i) {
        if (ld_dev(flag) != 0u) break;
        if (i >= kSpinLimit) {
            set_error(a, kErrSpin);
            break;
        }
        __builtin_amdgcn_s_sleep(4);
    }
    drain_memory();
}

// Wait until row `rid` has published its token; returns it.
__device__ int wait_token(const RaceArgs& a, int rid) {
    wait_nonzero(a, (const uint32_t*)(a.ws + a.L.flag) + rid);
    return ld_dev((const int32_t*)(a.ws + a.L.tok) + rid);
}

// ---------------------------------------------------------------- logits access

template <bool BF16>
__device__ __forceinline__ float load_logit(const unsigned char* row, int v) {
    if constexpr (BF16)
        return __uint_as_float((uint32_t)((const uint16_t*)row)[v] << 16);
    else
        return ((const float*)row)[v];
}

// 8 consecutive logits starting at `base` (-inf past V).
template <bool BF16, bool VEC>
__device__ __forceinline__ void load8(const unsigned char* row, int V, int base, float (&x)[8]) {
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
        for (int i = 0; i < 8; ++i) x[i] = (base + i < V) ? load_logit<BF16>(row, base + i) : -INFINITY;
    }
}

// ---------------------------------------------------------------- streaming pass

__device__ __forceinline__ void lse_combine(float& m, float& s, float om, float os) {
    const float mn = fmaxf(m, om);
    if (mn == -INFINITY) return;
    s = (m == -INFINITY ? 0.f : s * __builtin_amdgcn_exp2f(m - mn)) +
        (om == -INFINITY ? 0.f : os * __builtin_amdgcn_exp2f(om - mn));
    m = mn;
}

// One 32 KiB segment: group maxima -> gmax_row, (max, sum) of exp2(l * log2e / T) -> part_row[seg].
template <bool BF16, bool VEC>
__device__ void stream_segment(const RaceArgs& a, const Row& r, int seg, Shared& sm) {
    constexpr int NU = BF16 ? 8 : 4;  // 8-token units per lane
    const int tid = threadIdx.x;
    const int V = a.V;
    const int seg0 = seg * (BF16 ? kSegTokensBf16 : kSegTokensF32);
    float* gmax_row = (float*)(a.ws + a.L.gmax) + (size_t)r.row_id * a.L.ng;
    const float c2 = r.invT * 1.4426950408889634f;
    float x[NU][8];
#pragma unroll
    for (int q = 0; q < NU; ++q) load8<BF16, VEC>(r.ptr, V, seg0 + 8 * (q * kBlock + tid), x[q]);
    float mrun = -INFINITY, srun = 0.f;
#pragma unroll
    for (int q = 0; q < NU; ++q) {
        const int base = seg0 + 8 * (q * kBlock + tid);
        float um = fmaxf(fmaxf(fmaxf(x[q][0], x[q][1]), fmaxf(x[q][2], x[q][3])),
                         fmaxf(fmaxf(x[q][4], x[q][5]), fmaxf(x[q][6], x[q][7])));
        const float g = row16_max(um);
        if ((tid & 15) == 0 && base < V) st_dev(gmax_row + (base >> 7), g);
        const float mn = fmaxf(mrun, um * c2);
        if (mn != -INFINITY) {
            float acc = (mrun == -INFINITY) ? 0.f : srun * __builtin_amdgcn_exp2f(mrun - mn);
#pragma unroll
            for (int i = 0; i < 8; ++i) acc += __builtin_amdgcn_exp2f(fmaf(x[q][i], c2, -mn));
            srun = acc;
            mrun = mn;
        }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        const float om = __shfl_xor(mrun, off);
        const float os = __shfl_xor(srun, off);
        lse_combine(mrun, srun, om, os);
    }
    const int wave = tid >> 6;
    if ((tid & 63) == 0) {
        sm.red_a[wave] = mrun;
        sm.red_b[wave] = srun;
    }
    __syncthreads();
    if (tid == 0) {
        float m = sm.red_a[0], s = sm.red_b[0];
        for (int w = 1; w < kBlock / 64; ++w) lse_combine(m, s, sm.red_a[w], sm.red_b[w]);
        unsigned long long* part = (unsigned long long*)(a.ws + a.L.part) + (size_t)r.row_id * a.L.nseg;
        st_dev(part + seg, ((unsigned long long)__float_as_uint(s) << 32) | __float_as_uint(m));
    }
}

// ---------------------------------------------------------------- race search

__device__ __forceinline__ float current_threshold(Shared& sm) {
    return ordered_value(__hip_atomic_load(&sm.best_key, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP)) +
           kMargin;
}

__device__ __forceinline__ void push_node(Node* list, int* count, int cap, uint32_t id, float m, uint32_t p,
                                          const RaceArgs& a) {
    const int i = atomicAdd(count, 1);
    if (i < cap) list[i] = Node{id, m, p};
}

__device__ __forceinline__ void push_candidate(Shared& sm, const RaceArgs& a, int v, int j, float s) {
    const int i = atomicAdd(&sm.n_cand, 1);
    if (i < kCandCap) {
        sm.cand_v[i] = v;
        sm.cand_j[i] = j;
        sm.cand_s[i] = s;
    } else {
        set_error(a, kErrCand);
    }
}

// Evaluate chunk c (8 tokens) of a listed group for one slot.  The 16 lanes of a
// DPP row hold the 16 chunks of one group entry; the entry-level test is uniform
// over the row, and every lane of the row reaches the row minimum below, so only
// tokens within the margin of the group's best score become candidates (any
// token within the margin of the final best is within the margin of its group's).
template <bool BF16, bool VEC, int LAYOUT>
__device__ void eval_chunk(const RaceArgs& a, const Row& r, Shared& sm, const float* gm, const Node nd, int c,
                           uint32_t k0, uint32_t k1) {
    const uint32_t slot = nd.id >> 20;
    const uint32_t g = nd.id & 0xFFFFFu;
    const uint32_t V = (uint32_t)a.V;
    const float thr = current_threshold(sm);
    if (LAYOUT == 0 && ln_f32(nd.m) - gm[g] * r.invT > thr) return;
    if (LAYOUT == 1 && kLnClockFloor - gm[g] * r.invT > thr) return;
    const uint32_t base = g * kGroupTokens + (uint32_t)c * 8u;
    float sc[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) sc[i] = INFINITY;
    if (base < V) {
        float x[8];
        load8<BF16, VEC>(r.ptr, (int)V, (int)base, x);
        if constexpr (LAYOUT == 0) {
            const uint32_t chunk = g * 16u + (uint32_t)c;
            float mc;
            uint32_t pc;
            child_min_f32(nd.m, nd.p, 1, chunk, base, node_end(kShift1, chunk, V), slot, k0, k1, mc, pc);
            const float cmax =
                fmaxf(fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3])), fmaxf(fmaxf(x[4], x[5]), fmaxf(x[6], x[7])));
            if (ln_f32(mc) - cmax * r.invT <= thr) {
                const Words w0 = philox(chunk, slot, 8u, kDomainTree, k0, k1);
                const Words w1 = philox(chunk, slot, 9u, kDomainTree, k0, k1);
                const uint32_t ws[8] = {w0.w0, w0.w1, w0.w2, w0.w3, w1.w0, w1.w1, w1.w2, w1.w3};
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    const uint32_t v = base + (uint32_t)i;
                    if (v < V && x[i] != -INFINITY) {
                        const float E = (v == pc) ? mc : mc + exp1_f32(ws[i]);
                        sc[i] = ln_f32(E) - x[i] * r.invT;
                    }
                }
            }
        } else {
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                bool any = false;
#pragma unroll
                for (int i = 4 * h; i < 4 * h + 4; ++i)
                    any |= (base + (uint32_t)i < V) && (kLnClockFloor - x[i] * r.invT <= thr);
                if (!any) continue;
                const Words w = philox((base >> 2) + (uint32_t)h, slot, 0u, kDomainFlat, k0, k1);
                const uint32_t ws[4] = {w.w0, w.w1, w.w2, w.w3};
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const uint32_t v = base + (uint32_t)(4 * h + i);
                    const float xv = x[4 * h + i];
                    if (v < V && xv != -INFINITY) sc[4 * h + i] = ln_f32(exp1_f32(ws[i])) - xv * r.invT;
                }
            }
        }
    }
    float lm = sc[0];
#pragma unroll
    for (int i = 1; i < 8; ++i) lm = fminf(lm, sc[i]);
    const float rm = row16_min(lm);
    if (!(rm <= thr) || rm == INFINITY) return;
    if (lm == rm) atomicMin(&sm.best_key, ordered_key(rm));
    const float lim = fminf(thr, rm + kMargin);
#pragma unroll
    for (int i = 0; i < 8; ++i)
        if (sc[i] <= lim && sc[i] < INFINITY) push_candidate(sm, a, (int)(base + (uint32_t)i), (int)slot, sc[i]);
}

// Evaluate every listed group (16 lanes per group, 16 groups per pass), then empty the list.
template <bool BF16, bool VEC, int LAYOUT>
__device__ void flush_groups(const RaceArgs& a, const Row& r, Shared& sm, const float* gm, uint32_t k0,
                             uint32_t k1) {
    const int tid = threadIdx.x;
    const int n = min(sm.n_l2, kL2Cap);
    for (int base = 0; base < n; base += kBlock / 16) {
        const int e = base + (tid >> 4);
        if (e < n) eval_chunk<BF16, VEC, LAYOUT>(a, r, sm, gm, sm.l2[e], tid & 15, k0, k1);
        __syncthreads();
        if (tid == 0 && sm.n_cand > kCandCap / 2) {
            // keep only candidates still within the margin of the best score
            const float lim = ordered_value(sm.best_key) + kMargin;
            const int nc = min(sm.n_cand, kCandCap);
            int o = 0;
            for (int i = 0; i < nc; ++i)
                if (sm.cand_s[i] <= lim) {
                    sm.cand_v[o] = sm.cand_v[i];
                    sm.cand_j[o] = sm.cand_j[i];
                    sm.cand_s[o] = sm.cand_s[i];
                    ++o;
                }
            sm.n_cand = o;
        }
        __syncthreads();
    }
    if (tid == 0) sm.n_l2 = 0;
    __syncthreads();
}

// Expand listed level-3 nodes into level-2 groups (tree layout), evaluating groups as the list fills.
template <bool BF16, bool VEC>
__device__ void flush_l3(const RaceArgs& a, const Row& r, Shared& sm, const float* gm, uint32_t k0, uint32_t k1) {
    const int tid = threadIdx.x;
    const int n = min(sm.n_l3, kL3Cap) * 16;
    const uint32_t V = (uint32_t)a.V;
    for (int base = 0; base < n; base += kBlock) {
        // Every thread reads the list count before any thread of this pass can push
        // (otherwise waves could disagree on calling the barrier-bearing flush).
        const bool flush = sm.n_l2 > 0;
        __syncthreads();
        if (flush) flush_groups<BF16, VEC, 0>(a, r, sm, gm, k0, k1);
        const int e = base + tid;
        if (e < n) {
            const Node pa = sm.l3[e >> 4];
            const uint32_t g = (pa.id & 0xFFFFFu) * 16u + (uint32_t)(e & 15);
            const uint32_t cs = g << kShift2;
            if (cs < V) {
                const uint32_t slot = pa.id >> 20;
                float m;
                uint32_t p;
                child_min_f32(pa.m, pa.p, 2, g, cs, node_end(kShift2, g, V), slot, k0, k1, m, p);
                if (ln_f32(m) - gm[g] * r.invT <= current_threshold(sm))
                    push_node(sm.l2, &sm.n_l2, kL2Cap, (slot << 20) | g, m, p, a);
            }
        }
        __syncthreads();
    }
    if (sm.n_l2 > 0) flush_groups<BF16, VEC, 0>(a, r, sm, gm, k0, k1);
    __syncthreads();
    if (tid == 0) sm.n_l3 = 0;
    __syncthreads();
}

// Lexicographic minimum of (score, token, slot) over the workgroup.
__device__ __forceinline__ bool lex_less(double s, int v, int j, double s2, int v2, int j2) {
    return s < s2 || (s == s2 && (v < v2 || (v == v2 && j < j2)));
}

template <bool BF16, bool VEC, int LAYOUT>
__device__ void race(const RaceArgs& a, const Row& r, Shared& sm, const float* gm, uint32_t k0, uint32_t k1) {
    const int tid = threadIdx.x;
    const uint32_t V = (uint32_t)a.V;
    const int ng = a.L.ng;
    const int ns = r.nslots;
    if (tid == 0) {
        sm.n_l4 = sm.n_l3 = sm.n_l2 = sm.n_cand = 0;
        sm.best_key = ordered_key(INFINITY);
    }
    __syncthreads();

    // (A) threshold from the group holding the row maximum, for every slot.
    if (tid < ns && sm.gstar >= 0 && sm.gstar < ng) {
        const uint32_t slot = (uint32_t)(r.slot0 + tid);
        const uint32_t g = (uint32_t)sm.gstar;
        float m = 0.f;
        uint32_t p = 0u;
        if (LAYOUT == 0) {
            root_min_f32(V, slot, k0, k1, m, p);
            const int sh[3] = {kShift4, kShift3, kShift2};
#pragma unroll
            for (int l = 0; l < 3; ++l) {
                const uint32_t i = (g << kShift2) >> sh[l];
                child_min_f32(m, p, 4 - l, i, node_start(sh[l], i), node_end(sh[l], i, V), slot, k0, k1, m, p);
            }
        }
        sm.l2[tid] = Node{(slot << 20) | g, m, p};
    }
    if (tid == 0) sm.n_l2 = (sm.gstar >= 0 && sm.gstar < ng) ? ns : 0;
    __syncthreads();
    flush_groups<BF16, VEC, LAYOUT>(a, r, sm, gm, k0, k1);

    if constexpr (LAYOUT == 0) {
        // (B) tree descent: roots -> level 4 -> level 3 -> level 2 groups.
        if (tid < ns) root_min_f32(V, (uint32_t)(r.slot0 + tid), k0, k1, sm.root_m[tid], sm.root_p[tid]);
        __syncthreads();
        const int n4 = (int)((V + (1u << kShift4) - 1) >> kShift4);
        for (int base = 0; base < ns * n4; base += kBlock) {
            const int e = base + tid;
            if (e < ns * n4) {
                const int j = e / n4;
                const uint32_t i4 = (uint32_t)(e % n4);
                const uint32_t slot = (uint32_t)(r.slot0 + j);
                float m;
                uint32_t p;
                child_min_f32(sm.root_m[j], sm.root_p[j], 4, i4, node_start(kShift4, i4), node_end(kShift4, i4, V),
                              slot, k0, k1, m, p);
                if (ln_f32(m) - sm.m4[i4] * r.invT <= current_threshold(sm))
                    push_node(sm.l4, &sm.n_l4, kL4Cap, (slot << 20) | i4, m, p, a);
            }
        }
        __syncthreads();
        const int n3tot = min(sm.n_l4, kL4Cap) * 16;
        for (int base = 0; base < n3tot; base += kBlock) {
            const bool flush = sm.n_l3 + kBlock > kL3Cap;
            __syncthreads();
            if (flush) flush_l3<BF16, VEC>(a, r, sm, gm, k0, k1);
            const int e = base + tid;
            if (e < n3tot) {
                const Node pa = sm.l4[e >> 4];
                const uint32_t i3 = (pa.id & 0xFFFFFu) * 16u + (uint32_t)(e & 15);
                const uint32_t cs = i3 << kShift3;
                if (cs < V) {
                    const uint32_t slot = pa.id >> 20;
                    float m;
                    uint32_t p;
                    child_min_f32(pa.m, pa.p, 3, i3, cs, node_end(kShift3, i3, V), slot, k0, k1, m, p);
                    if (ln_f32(m) - sm.m3[i3] * r.invT <= current_threshold(sm))
                        push_node(sm.l3, &sm.n_l3, kL3Cap, (slot << 20) | i3, m, p, a);
                }
            }
            __syncthreads();
        }
        flush_l3<BF16, VEC>(a, r, sm, gm, k0, k1);
    } else {
        // (B) flat clocks: every (group, slot) whose floor bound can win.
        const int tot = ng * ns;
        for (int base = 0; base < tot; base += kBlock) {
            const bool flush = sm.n_l2 > 0;
            __syncthreads();
            if (flush) flush_groups<BF16, VEC, 1>(a, r, sm, gm, k0, k1);
            const int e = base + tid;
            if (e < tot) {
                const int g = e / ns;
                const uint32_t slot = (uint32_t)(r.slot0 + e % ns);
                if (kLnClockFloor - gm[g] * r.invT <= current_threshold(sm))
                    push_node(sm.l2, &sm.n_l2, kL2Cap, (slot << 20) | (uint32_t)g, 0.f, 0u, a);
            }
            __syncthreads();
        }
        flush_groups<BF16, VEC, 1>(a, r, sm, gm, k0, k1);
    }

    // (C) exact decision among the candidates within the margin of the best.
    const float best = ordered_value(sm.best_key);
    const int nc = min(sm.n_cand, kCandCap);
    double bs = INFINITY;
    int bv = 0x7FFFFFFF, bj = 0x7FFFFFFF;
    for (int i = tid; i < nc; i += kBlock) {
        if (sm.cand_s[i] > best + kMargin) continue;
        const int v = sm.cand_v[i], j = sm.cand_j[i];
        const double E = LAYOUT == 0 ? tree_clock_f64(V, (uint32_t)j, (uint32_t)v, k0, k1)
                                     : flat_clock_f64((uint32_t)j, (uint32_t)v, k0, k1);
        const double s = log(E) - (double)load_logit<BF16>(r.ptr, v) / (double)r.T;
        if (lex_less(s, v, j, bs, bv, bj)) {
            bs = s;
            bv = v;
            bj = j;
        }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        const double os = __shfl_xor(bs, off);
        const int ov = __shfl_xor(bv, off), oj = __shfl_xor(bj, off);
        if (lex_less(os, ov, oj, bs, bv, bj)) {
            bs = os;
            bv = ov;
            bj = oj;
        }
    }
    if ((tid & 63) == 0) {
        sm.red_s[tid >> 6] = bs;
        sm.red_v[tid >> 6] = bv;
        sm.red_j[tid >> 6] = bj;
    }
    __syncthreads();
    if (tid == 0) {
        for (int w = 1; w < kBlock / 64; ++w)
            if (lex_less(sm.red_s[w], sm.red_v[w], sm.red_j[w], bs, bv, bj)) {
                bs = sm.red_s[w];
                bv = sm.red_v[w];
                bj = sm.red_j[w];
            }
        sm.win_token = (bs < INFINITY) ? bv : -1;
        sm.win_slot = (bs < INFINITY) ? bj : -1;
    }
    __syncthreads();
}

// ---------------------------------------------------------------- walk

__device__ void walk(const RaceArgs& a, int b) {
    const int K = a.K, G = a.gamma;
    const int32_t* tok = (const int32_t*)(a.ws + a.L.tok);
    uint32_t act = K >= 32 ? 0xFFFFFFFFu : ((1u << K) - 1u);
    int tau = 0;
    bool done = false;
    for (int s = 0; s < G && !done; ++s) {
        const int kk = __ffs((int)act) - 1;
        const int y = ld_dev(tok + target_row_id(a, b, kk, s));
        a.out_tokens[(size_t)b * (G + 1) + s] = y;
        tau = s + 1;
        if (y < 0) {
            done = true;
            break;
        }
        uint32_t na = 0u;
        for (int k = 0; k < K; ++k)
            if (((act >> k) & 1u) && ld_dev(a.draft_tokens + ((size_t)b * K + k) * G + s) == y) na |= 1u << k;
        if (!na) {
            done = true;
            break;
        }
        act = na;
    }
    if (!done) {
        const int kk = __ffs((int)act) - 1;
        a.out_tokens[(size_t)b * (G + 1) + G] = ld_dev(tok + target_row_id(a, b, kk, G));
        tau = G + 1;
    }
    for (int s = tau; s <= G; ++s) a.out_tokens[(size_t)b * (G + 1) + s] = -1;
    a.out_len[b] = tau;
}

// ---------------------------------------------------------------- row finisher

template <bool BF16, bool VEC, int LAYOUT>
__device__ void finish_row(const RaceArgs& a, const Row& r, Shared& sm, float* gm) {
    const int tid = threadIdx.x;
    const int ng = a.L.ng;
    const int n3 = (ng + 15) / 16, n4 = (n3 + 15) / 16;
    const float* gsrc = (const float*)(a.ws + a.L.gmax) + (size_t)r.row_id * ng;
    for (int g = tid; g < ng; g += kBlock) gm[g] = ld_dev(gsrc + g);
    if (tid == 0) {
        // LSE from the segment partials (log2 units), merged in double.
        const unsigned long long* part = (const unsigned long long*)(a.ws + a.L.part) + (size_t)r.row_id * a.L.nseg;
        double M = -INFINITY, S = 0.0;
        for (int i = 0; i < a.L.nseg; ++i) {
            const unsigned long long bits = ld_dev(part + i);
            const double pm = (double)__uint_as_float((uint32_t)bits), ps = (double)__uint_as_float((uint32_t)(bits >> 32));
            if (pm == -INFINITY) continue;
            if (pm > M) {
                S = (M == -INFINITY ? 0.0 : S * exp2(M - pm)) + ps;
                M = pm;
            } else {
                S += ps * exp2(pm - M);
            }
        }
        const double lse = M == -INFINITY ? -INFINITY : (M + log2(S)) * 0.69314718055994530942;
        if (r.kind == 0) {
            if (a.draft_lse) a.draft_lse[((size_t)r.b * a.K + r.k) * a.gamma + r.s] = (float)lse;
        } else if (a.target_lse) {
            const size_t o = a.target_rows == 1 ? (size_t)r.b * (a.gamma + 1) + r.s
                                                : ((size_t)r.b * a.K + r.k) * (a.gamma + 1) + r.s;
            a.target_lse[o] = (float)lse;
        }
        // Context window: last m tokens of prefix || path tokens before depth s.
        for (int i = 0; i < a.m; ++i) {
            const int idx = r.s + i;  // index into prefix (m tokens) || path (s tokens)
            int tk;
            if (idx < a.m) {
                tk = a.prefix[(size_t)r.b * a.m + idx];
            } else {
                const int d = idx - a.m;  // path depth
                if (r.kind == 1 && a.target_rows == 1) {
                    tk = wait_token(a, target_row_id(a, r.b, 0, d));
                } else if (a.s_count > 0 && d >= a.s_begin) {
                    tk = wait_token(a, draft_row_id(a, r.b, r.k, d));
                } else {
                    tk = a.draft_tokens[((size_t)r.b * a.K + r.k) * a.gamma + d];
                }
            }
            sm.window[i] = tk;
        }
        uint32_t k0, k1;
        context_key(a.key, a.start_pos[r.b] + r.s, sm.window, a.m, k0, k1);
        sm.kappa0 = k0;
        sm.kappa1 = k1;
    }
    __syncthreads();
    for (int t = tid; t < n3; t += kBlock) {
        float mx = -INFINITY;
        for (int g = 16 * t; g < min(ng, 16 * t + 16); ++g) mx = fmaxf(mx, gm[g]);
        sm.m3[t] = mx;
    }
    // argmax group (lowest index among equal maxima)
    float bvv = -INFINITY;
    int bi = 0x7FFFFFFF;
    for (int g = tid; g < ng; g += kBlock)
        if (gm[g] > bvv) {
            bvv = gm[g];
            bi = g;
        }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        const float ov = __shfl_xor(bvv, off);
        const int oi = __shfl_xor(bi, off);
        if (ov > bvv || (ov == bvv && oi < bi)) {
            bvv = ov;
            bi = oi;
        }
    }
    if ((tid & 63) == 0) {
        sm.red_a[tid >> 6] = bvv;
        sm.red_v[tid >> 6] = bi;
    }
    __syncthreads();
    if (tid < n4) {
        float mx = -INFINITY;
        for (int t = 16 * tid; t < min(n3, 16 * tid + 16); ++t) mx = fmaxf(mx, sm.m3[t]);
        sm.m4[tid] = mx;
    }
    if (tid == 0) {
        for (int w = 1; w < kBlock / 64; ++w)
            if (sm.red_a[w] > bvv || (sm.red_a[w] == bvv && sm.red_v[w] < bi)) {
                bvv = sm.red_a[w];
                bi = sm.red_v[w];
            }
        sm.rowmax = bvv;
        sm.gstar = bi;
    }
    __syncthreads();
    const uint32_t k0 = sm.kappa0, k1 = sm.kappa1;
    if (sm.rowmax == -INFINITY) {
        if (tid == 0) {
            sm.win_token = -1;
            sm.win_slot = -1;
        }
        __syncthreads();
    } else {
        race<BF16, VEC, LAYOUT>(a, r, sm, gm, k0, k1);
    }
    if (tid == 0) {
        const int y = sm.win_token;
        if (r.kind == 0) {
            st_dev(a.draft_tokens + ((size_t)r.b * a.K + r.k) * a.gamma + r.s, y);
        } else if (a.target_tokens) {
            const size_t o = a.target_rows == 1 ? (size_t)r.b * (a.gamma + 1) + r.s
                                                : ((size_t)r.b * a.K + r.k) * (a.gamma + 1) + r.s;
            a.target_tokens[o] = y;
        }
        st_dev((int32_t*)(a.ws + a.L.tok) + r.row_id, y);
        drain_memory();
        st_dev((uint32_t*)(a.ws + a.L.flag) + r.row_id, 1u);
        if (a.target_rows > 0) {
            uint32_t* sc = (uint32_t*)(a.ws + a.L.seq_cnt) + r.b;
            const uint32_t old = __hip_atomic_fetch_add(sc, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if ((int)old + 1 == a.seq_rows) {
                drain_memory();
                walk(a, r.b);
            }
        }
    }
}

// ---------------------------------------------------------------- kernel

template <bool BF16, bool VEC, int LAYOUT>
__global__ __launch_bounds__(kBlock) void race_kernel(RaceArgs a) {
    extern __shared__ __align__(16) unsigned char smem_raw[];
    Shared& sm = *reinterpret_cast<Shared*>(smem_raw);
    float* gm = reinterpret_cast<float*>(smem_raw + ((sizeof(Shared) + 15) & ~(size_t)15));
    const int tid = threadIdx.x;
    uint32_t* ctrl = ctrl_of(a);
    const size_t esize = BF16 ? 2 : 4;
    const int D = a.B * a.K * a.gamma;
    // Ticket 0 clears this call's row counters, flags and sequence counters (their
    // placement depends on the call's shape, so a previous call with another shape
    // may have left data there); every workgroup waits for that clear before its
    // first counter update.  Tickets 1.. are the work items.
    bool cleared = false;
    for (;;) {
        if (tid == 0) sm.item = (int)atomicAdd(ctrl, 1u) - 1;
        __syncthreads();
        const int item = sm.item;
        if (item >= a.n_items) break;
        if (item < 0) {
            uint32_t* base = (uint32_t*)(a.ws + a.L.row_cnt);
            const size_t n = (a.L.ctrl_end - a.L.row_cnt) / 4;
            for (size_t i = tid; i < n; i += kBlock) st_dev(base + i, 0u);
            drain_memory();
            __syncthreads();
            if (tid == 0) st_dev(ctrl + 4, 1u);
            cleared = true;
            continue;
        }
        int d = 0;
        while (d + 1 < a.n_depth && item >= a.depth_first[d + 1]) ++d;
        const int local = item - a.depth_first[d];
        const int rl = local / a.L.nseg, seg = local % a.L.nseg;
        Row r;
        r.s = d;
        if (rl < a.depth_nd[d]) {
            r.kind = 0;
            r.b = rl / a.K;
            r.k = rl % a.K;
            r.row_id = (r.b * a.K + r.k) * a.gamma + d;
            r.ptr = (const unsigned char*)a.draft_logits +
                    (((size_t)r.b * a.K + r.k) * a.s_count + (size_t)(d - a.s_begin)) * (size_t)a.V * esize;
            r.slot0 = r.k;
            r.nslots = 1;
            r.invT = a.inv_T_draft;
            r.T = a.T_draft;
        } else {
            const int rt = rl - a.depth_nd[d];
            r.kind = 1;
            size_t off;
            if (a.target_rows == 1) {
                r.b = rt;
                r.k = 0;
                r.row_id = D + r.b * (a.gamma + 1) + d;
                off = (size_t)r.b * (a.gamma + 1) + d;
            } else {
                r.b = rt / a.K;
                r.k = rt % a.K;
                r.row_id = D + (r.b * a.K + r.k) * (a.gamma + 1) + d;
                off = ((size_t)r.b * a.K + r.k) * (a.gamma + 1) + d;
            }
            r.ptr = (const unsigned char*)a.target_logits + off * (size_t)a.V * esize;
            r.slot0 = 0;
            r.nslots = a.K;
            r.invT = a.inv_T_target;
            r.T = a.T_target;
        }
        stream_segment<BF16, VEC>(a, r, seg, sm);
        drain_memory();
        __syncthreads();
        if (tid == 0) {
            if (!cleared) wait_nonzero(a, ctrl + 4);
            uint32_t* rc = (uint32_t*)(a.ws + a.L.row_cnt) + r.row_id;
            const uint32_t old = __hip_atomic_fetch_add(rc, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            drain_memory();
            sm.fin = ((int)old == a.L.nseg - 1);
        }
        cleared = true;
        __syncthreads();
        if (sm.fin) finish_row<BF16, VEC, LAYOUT>(a, r, sm, gm);
        __syncthreads();
    }
    // The last workgroup to leave resets the fixed header words for the next call.
    if (tid == 0) {
        drain_memory();
        const uint32_t old = __hip_atomic_fetch_add(ctrl + 1, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (old == gridDim.x - 1) {
            st_dev(ctrl + 0, 0u);
            st_dev(ctrl + 1, 0u);
            st_dev(ctrl + 4, 0u);
        }
    }
}

template <bool BF16, bool VEC, int LAYOUT>
hipError_t launch_one(const RaceArgs& a, hipStream_t stream) {
    const size_t smem = ((sizeof(Shared) + 15) & ~(size_t)15) + (size_t)a.L.ng * sizeof(float);
    auto fn = race_kernel<BF16, VEC, LAYOUT>;
    int per_cu = 0;
    hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kBlock, smem);
    if (e != hipSuccess) return e;
    int dev = 0, cus = 0;
    if ((e = hipGetDevice(&dev)) != hipSuccess) return e;
    if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess) return e;
    if (per_cu < 1) per_cu = 1;
    long grid = (long)per_cu * cus;
    if (grid > a.n_items) grid = a.n_items;
    if (grid < 1) grid = 1;
    hipLaunchKernelGGL(fn, dim3((unsigned)grid), dim3(kBlock), smem, stream, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_race(const RaceArgs& a, bool bf16, bool vec, int layout, hipStream_t stream) {
    if (bf16) {
        if (vec) return layout == 0 ? launch_one<true, true, 0>(a, stream) : launch_one<true, true, 1>(a, stream);
        return layout == 0 ? launch_one<true, false, 0>(a, stream) : launch_one<true, false, 1>(a, stream);
    }
    if (vec) return layout == 0 ? launch_one<false, true, 0>(a, stream) : launch_one<false, true, 1>(a, stream);
    return layout == 0 ? launch_one<false, false, 0>(a, stream) : launch_one<false, false, 1>(a, stream);
}

size_t race_shared_bytes(int ng) { return ((sizeof(Shared) + 15) & ~(size_t)15) + (size_t)ng * sizeof(float); }

}  // namespace psd
