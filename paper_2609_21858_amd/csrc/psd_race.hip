// psd_race.hip -- fused draft + verify kernel of the keyed Poisson race (gfx950).
//
// One persistent kernel per call.  Rows are numbered depth-major (all rows of
// depth 0, then depth 1, ...) and dealt round-robin to up to eight work queues,
// one per XCD (workgroup w serves queue w mod 8), so the ticket counters are not
// one contended atomic; a queue hands out its rows' 32 KiB segments in order, so
// every row a race depends on is handed out before the rows that depend on it.
//
// Per segment (key-independent, HBM-streaming): coalesced 16-byte non-temporal
// loads, the online log-sum-exp partial (sum of exp2 relative to the segment
// maximum) and the maximum logit of every 128-token group.  Each value is published
// as one 64-bit slot tagged with the call's epoch, so nothing waits for stores to
// drain and nothing is cleared between calls.  The workgroup that holds a row's
// last segment becomes the row's finisher: it gathers the row's slots and does all
// key-independent work (block maxima, top groups, LSE), then folds the context key
// (waiting only for the newest context token), runs the keyed race, publishes the
// winner and -- for the last row of a sequence -- walks the block.
//
// The race (TREE clocks): the argmax tokens of four top groups give achievable
// scores; a level-by-level descent then expands only nodes whose lower bound
// ln(min clock of the node) - max logit / T can still beat the best score; a
// child's minimum is never below its parent's, so the parent's minimum bounds a
// child before its own draw.  Only the 128-token groups that survive are re-read.
// FLAT clocks: every group whose floor bound ln(clock floor) - max logit / T can
// win is re-read and its surviving tokens draw their Philox word.
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

#include <mutex>

#include "psd_device.hpp"
#include "psd_launch.hpp"
#include "psd_layout.hpp"

namespace psd {

namespace {

constexpr int kInit = 8;                   // seed tokens of a race (segment top tokens)
constexpr int kL3Cap = 512;
constexpr int kL2Cap = 512;
constexpr int kRowEntries = 2;             // group entries per 16-lane row and evaluation pass
constexpr int kCandCap = 256;
constexpr int kWorkCap = 2048;             // (level-3 node, group) items per prefilter round
constexpr int kRolePeriod = 11;            // workgroup roles: of every kRolePeriod blocks,
constexpr int kRoleFinish = 4;             // kRoleFinish finish rows and the others stream
constexpr int kHalfCap = 256;              // 4-token halves listed by one evaluation pass
constexpr int kPassGroups = 16 * kRowEntries;  // group entries of one evaluation pass
constexpr int kBuckets = 32;               // bound buckets of the group list's evaluation order
constexpr float kMargin = 1e-3f;           // float32 pruning / candidate margin (score units)
constexpr float kCutSlack = 1e-3f;         // slack of the per-token logit cut (score units)
constexpr uint32_t kErrSpin = 1u, kErrCand = 2u;

struct Node {
    uint32_t id;  // (slot << 20) | node index
    float m;      // float32 minimum clock of the node
    uint32_t p;   // token holding that minimum
};

// A 4-token half of a chunk that can still win: entry (local index), chunk, half
// and token mask packed in desc; cref 0 when the chunk needs its own minimum drawn
// (-1: the chunk holds the group minimum); its logits.
struct Half {
    uint32_t desc;  // entry << 9 | chunk << 5 | half << 4 | token mask (4 bits)
    int cref;
    float x[4];
};

struct Shared {
    float m3[256];
    float m4[16];
    int init_v[kInit];     // seed groups of the race (-1: none)
    int seed_tok[kInit];   // seed tokens of the race (-1: none)
    int stop[64];          // top group of every segment (-1: none)
    float part[64];        // LSE partial sum of every segment
    Node l3[kL3Cap];
    Node l2[kL2Cap];
    int cand_v[kCandCap];
    int cand_j[kCandCap];
    float cand_s[kCandCap];
    float cand_x[kCandCap];
    double red_s[kBlock / 64];
    int red_v[kBlock / 64];
    int red_j[kBlock / 64];
    float red_a[2][kBlock / 64];  // per-wave LSE partials of the streamed segment (by parity)
    float red_b[2][kBlock / 64];
    int n_l4, n_l3, n_l2, n_cand;
    int best_key;
    int tick[4];
    int ph_first[kMaxPhases], ph_depth[kMaxPhases], ph_nd[kMaxPhases];  // work-order phases
    uint32_t epoch;
    float gst[2][128];  // group maxima of the streamed segment (by parity)
    int win_token, win_slot;
    float rowmax;
    uint32_t kappa0, kappa1;
    uint32_t next0, next1;  // partial context key of the path's next depth
    int win[32];            // context tokens (own window, next depth's window)
    int key_min, key_max;   // (token, slot) range of the candidates near the best
    uint32_t err_local;       // error bits this workgroup recorded (it then publishes them with a release)
    uint16_t work[kWorkCap];  // compacted work items (level-3 list index * 16 + group)
    int n_work;
    uint32_t n_ev[2];                 // listed halves, per pass parity
    Half half[kHalfCap];
    // evaluation order of the group list (order_groups)
    float ord_wmin[kBlock / 64];          // per-wave smallest bound
    int ord_hist[kBuckets];               // entries per bound bucket
    int ord_bmin[kBuckets];               // smallest bound per bucket (ordered key)
    int ord_pass[(kL2Cap + kPassGroups - 1) / kPassGroups];  // bucket of each pass's first entry
};
static_assert(sizeof(Half) * kHalfCap >= sizeof(Node) * kL2Cap, "the reordering stages the group list in half[]");

// Dynamic LDS after Shared: the group maxima gm (ng floats, rounded up to 4), then
// the level-4 node list of a race (K slots x level-4 nodes; sized at launch).
__device__ __forceinline__ Node* level4_list(const float* gm, int ng) {
    return (Node*)(gm + ((ng + 3) & ~3));
}

struct Row {
    int kind;  // 0 draft, 1 target
    int b, k, s;
    int row_id;
    const unsigned char* ptr;
    int slot0, nslots;
    float invT;
    float T;
    float shift;  // the row's maximum logit: fp32 scores and bounds use (l - shift) / T
};

// Scaled logit (l - shift) / T of the race's fp32 scores and bounds.  Near the
// top of the row the subtraction is exact (Sterbenz), so the scaled value of every
// token that can still win is O(tens) and rounds to a few 1e-6 score units
// whatever the magnitude of l / T; tokens far below the maximum have scores far
// above the threshold, where rounding cannot change a decision.
__device__ __forceinline__ float scaled(const Row& r, float x) { return (x - r.shift) * r.invT; }

__device__ __forceinline__ uint32_t* ctrl_of(const RaceArgs& a) { return (uint32_t*)(a.ws + a.L.ctrl); }

// Errors of the running call; its last workgroup hands them to the sticky word and
// to the caller's status word.  The workgroup also notes them in LDS, so that its
// exit publishes them with a release (see the end of race_kernel).
__device__ __forceinline__ void set_error(const RaceArgs& a, uint32_t bit) {
    extern __shared__ __align__(16) unsigned char smem_raw[];
    __hip_atomic_fetch_or(ctrl_of(a) + kCtrlCallErrors, bit, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    atomicOr(&reinterpret_cast<Shared*>(smem_raw)->err_local, bit);
}

// Cross-workgroup slots are touched only with relaxed device-scope atomics, which
// are coherent across the XCDs without L2-wide write-back / invalidate; each slot
// carries its epoch, so a reader knows when the producer's value has landed.
template <typename T>
__device__ __forceinline__ void st_dev(T* p, T v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
template <typename T>
__device__ __forceinline__ T ld_dev(const T* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Bounded wait for a slot whose tag (high 32 bits) equals the epoch.  On timeout an
// error bit is recorded and the stale value is returned, so every wave terminates.
__device__ __forceinline__ uint64_t wait_slot(const RaceArgs& a, const uint64_t* p, uint32_t epoch) {
    uint64_t v = ld_dev(p);
    for (uint32_t i = 0; (uint32_t)(v >> 32) != epoch; ++i) {
        if (i >= a.spin_limit) {
            set_error(a, kErrSpin);
            break;
        }
        __builtin_amdgcn_s_sleep(2);
        v = ld_dev(p);
    }
    return v;
}

__device__ __forceinline__ int target_row_id(const RaceArgs& a, int b, int k, int s) {
    const int D = a.B * a.K * a.gamma;
    return a.target_rows == 1 ? D + b * (a.gamma + 1) + s : D + (b * a.K + k) * (a.gamma + 1) + s;
}

__device__ __forceinline__ int draft_row_id(const RaceArgs& a, int b, int k, int s) {
    return (b * a.K + k) * a.gamma + s;
}

__device__ __forceinline__ int wait_token(const RaceArgs& a, int rid, uint32_t epoch) {
    return (int)(uint32_t)wait_slot(a, (const uint64_t*)(a.ws + a.L.tok) + rid, epoch);
}

// Next work item of queue q (of nq): the queue's rows are R = q, q + nq, ... in
// depth-major order, each handed out segment by segment.  Returns n_items when the
// queue is exhausted.
__device__ __forceinline__ int take_item(const RaceArgs& a, int q, int nq) {
    const uint32_t t = atomicAdd(ctrl_of(a) + ctrl_queue(q), 1u);
    const uint32_t R = (uint32_t)q + (uint32_t)nq * (t / (uint32_t)a.L.nseg);
    return R >= (uint32_t)a.n_rows ? a.n_items : (int)(R * (uint32_t)a.L.nseg + t % (uint32_t)a.L.nseg);
}

// Next row of row queue q (of nq) for a finishing workgroup: rows R = q, q + nq, ...
// in work order.  Returns n_rows when the queue is exhausted.
__device__ __forceinline__ int take_row(const RaceArgs& a, int q, int nq) {
    const uint32_t t = atomicAdd(ctrl_of(a) + ctrl_queue(kMaxQueues + q), 1u);
    const uint32_t R = (uint32_t)q + (uint32_t)nq * t;
    return R >= (uint32_t)a.n_rows ? a.n_rows : (int)R;
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

// Raw 16-byte words of one 8-token unit (bf16: one word, float32: two); -inf past V.
template <bool BF16, bool VEC>
struct Unit {
    uint4 w[BF16 ? 1 : 2];
};

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <bool NT>
__device__ __forceinline__ uint4 ld16(const void* p) {
    if constexpr (NT) {
        const u32x4 v = __builtin_nontemporal_load((const u32x4*)p);
        return make_uint4(v.x, v.y, v.z, v.w);
    } else {
        return *(const uint4*)p;
    }
}

// Vector path: the address is clamped into the row (V * element size is a multiple
// of 16 bytes there), so every load is unconditional and the compiler can wait for
// them one by one; words past V are left for the caller to mask.  NT: streaming
// (non-temporal) loads for the single pass over the logits; re-reads of a few
// groups use ordinary loads.
template <bool BF16, bool VEC, bool NT = true>
__device__ __forceinline__ void load_unit(const unsigned char* row, int V, int base, Unit<BF16, VEC>& u) {
    if constexpr (VEC) {
        if constexpr (BF16) {
            u.w[0] = ld16<NT>((const uint16_t*)row + min(base, V - 8));
        } else {
            u.w[0] = ld16<NT>((const float*)row + min(base, V - 4));
            u.w[1] = ld16<NT>((const float*)row + min(base + 4, V - 4));
        }
    } else {
        float x[8];
        load8<BF16, false>(row, V, base, x);
        if constexpr (BF16) {
            uint32_t p[4];
#pragma unroll
            for (int i = 0; i < 4; ++i)
                p[i] = (__float_as_uint(x[2 * i]) >> 16) | (__float_as_uint(x[2 * i + 1]) & 0xFFFF0000u);
            u.w[0] = make_uint4(p[0], p[1], p[2], p[3]);
        } else {
            u.w[0] = make_uint4(__float_as_uint(x[0]), __float_as_uint(x[1]), __float_as_uint(x[2]), __float_as_uint(x[3]));
            u.w[1] = make_uint4(__float_as_uint(x[4]), __float_as_uint(x[5]), __float_as_uint(x[6]), __float_as_uint(x[7]));
        }
    }
}

template <bool BF16, bool VEC>
__device__ __forceinline__ void unpack_unit(const Unit<BF16, VEC>& u, float (&x)[8]) {
    if constexpr (BF16) {
        x[0] = bf16_lo(u.w[0].x); x[1] = bf16_hi(u.w[0].x); x[2] = bf16_lo(u.w[0].y); x[3] = bf16_hi(u.w[0].y);
        x[4] = bf16_lo(u.w[0].z); x[5] = bf16_hi(u.w[0].z); x[6] = bf16_lo(u.w[0].w); x[7] = bf16_hi(u.w[0].w);
    } else {
        x[0] = __uint_as_float(u.w[0].x); x[1] = __uint_as_float(u.w[0].y);
        x[2] = __uint_as_float(u.w[0].z); x[3] = __uint_as_float(u.w[0].w);
        x[4] = __uint_as_float(u.w[1].x); x[5] = __uint_as_float(u.w[1].y);
        x[6] = __uint_as_float(u.w[1].z); x[7] = __uint_as_float(u.w[1].w);
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

// Running maxima start at a finite sentinel, so that rescaling never meets inf - inf.
constexpr float kNegBig = -1e30f;

__device__ __forceinline__ void lse_merge_finite(float& m, float& s, float om, float os) {
    const float mn = fmaxf(m, om);
    s = s * __builtin_amdgcn_exp2f(m - mn) + os * __builtin_amdgcn_exp2f(om - mn);
    m = mn;
}

// One 32 KiB segment: the maximum logit of every 128-token group (16 lanes hold a
// group) and the segment's sum of exp2(l * log2e / T - M), M = log2e / T * (segment
// maximum).  Unless the workgroup is about to finish a row (which can wait on other
// workgroups), thread 0 takes its next ticket while the loads are in flight: a
// ticket held through such a wait would stall the rows that need that segment.
template <bool BF16>
constexpr int units_per_segment() {
    return BF16 ? 8 : 4;  // 2048-token units
}

// Issue the loads of one segment (one 8-token unit per thread and unit).
template <bool BF16, bool VEC>
__device__ __forceinline__ void issue_segment(const RaceArgs& a, const Row& r, int seg,
                                              Unit<BF16, VEC> (&u)[units_per_segment<BF16>()]) {
    constexpr int NU = units_per_segment<BF16>();
    const int seg0 = seg * (BF16 ? kSegTokensBf16 : kSegTokensF32);
#pragma unroll
    for (int q = 0; q < NU; ++q) load_unit<BF16, VEC>(r.ptr, a.V, seg0 + q * kBlock * 8 + 8 * threadIdx.x, u[q]);
}

// Consume a loaded segment: per-wave LSE partials and the maximum of every
// 128-token group, staged in LDS (parity p) for publish_segment.
template <bool BF16, bool VEC>
__device__ __forceinline__ void consume_segment(const RaceArgs& a, const Row& r, int seg, Shared& sm, int p,
                                                const Unit<BF16, VEC> (&u)[units_per_segment<BF16>()]) {
    constexpr int NU = units_per_segment<BF16>();
    constexpr int UT = kBlock * 8;
    const int tid = threadIdx.x, lane = tid & 63;
    const int V = a.V;
    const int seg0 = seg * (BF16 ? kSegTokensBf16 : kSegTokensF32);
    const float c2 = r.invT * 1.4426950408889634f;
    float mrun = kNegBig, srun = 0.f;
#pragma unroll
    for (int q = 0; q < NU; ++q) {
        float x[8];
        unpack_unit<BF16, VEC>(u[q], x);
        const int ub = seg0 + q * UT;
        if (ub + UT > V) {  // uniform: this unit reaches past the row
            const int base = ub + 8 * tid;
#pragma unroll
            for (int i = 0; i < 8; ++i)
                if (base + i >= V) x[i] = -INFINITY;
        }
        const float um = fmaxf(fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3])), fmaxf(fmaxf(x[4], x[5]), fmaxf(x[6], x[7])));
        const float g = row16_max(um);
        if ((lane & 15) == 0) sm.gst[p][q * 16 + (tid >> 4)] = g;
        const float mn = fmaxf(mrun, um * c2);
        float acc = srun * __builtin_amdgcn_exp2f(mrun - mn);
#pragma unroll
        for (int i = 0; i < 8; ++i) acc += __builtin_amdgcn_exp2f(fmaf(x[i], c2, -mn));
        srun = acc;
        mrun = mn;
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) lse_merge_finite(mrun, srun, __shfl_xor(mrun, off), __shfl_xor(srun, off));
    if (lane == 0) {
        sm.red_a[p][tid >> 6] = mrun;
        sm.red_b[p][tid >> 6] = srun;
    }
}

// Publish a consumed segment (after a barrier): one 64-bit slot per group and per
// 2048-token block, written by consecutive lanes, the segment's top group and its
// LSE partial.
template <bool BF16>
__device__ __forceinline__ void publish_segment(const RaceArgs& a, int row_id, int seg, Shared& sm, int p) {
    constexpr int NU = units_per_segment<BF16>();
    const int tid = threadIdx.x, lane = tid & 63;
    const int seg0 = seg * (BF16 ? kSegTokensBf16 : kSegTokensF32);
    const uint64_t ep = (uint64_t)sm.epoch << 32;
    const int g0 = seg0 >> 7;
    if (tid < NU * 16 && g0 + tid < a.L.ng) {
        uint64_t* gslot = (uint64_t*)(a.ws + a.L.gmax) + (size_t)row_id * a.L.ng;
        st_dev(gslot + g0 + tid, ep | __float_as_uint(sm.gst[p][tid]));
    } else if (tid >= 128 && tid < 128 + NU && (seg0 >> 11) + (tid - 128) < a.L.n3) {
        const int q = tid - 128;
        float mx = sm.gst[p][16 * q];
#pragma unroll
        for (int i = 1; i < 16; ++i) mx = fmaxf(mx, sm.gst[p][16 * q + i]);
        uint64_t* m3slot = (uint64_t*)(a.ws + a.L.m3) + (size_t)row_id * a.L.n3;
        st_dev(m3slot + (seg0 >> 11) + q, ep | __float_as_uint(mx));
    }
    if (tid < 64) {
        // the segment's top group: its largest group, lowest index on ties
        float bv = lane < NU * 16 ? sm.gst[p][lane] : -INFINITY;
        int bi = lane;
        if (lane + 64 < NU * 16 && sm.gst[p][lane + 64] > bv) {
            bv = sm.gst[p][lane + 64];
            bi = lane + 64;
        }
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) {
            const float ov = __shfl_xor(bv, off);
            const int oi = __shfl_xor(bi, off);
            if (ov > bv || (ov == bv && oi < bi)) {
                bv = ov;
                bi = oi;
            }
        }
        if (lane == 0) {
            uint64_t* stop = (uint64_t*)(a.ws + a.L.stop) + (size_t)row_id * a.L.nseg;
            st_dev(stop + seg, ep | (uint32_t)(bv == -INFINITY ? -1 : g0 + bi));
        }
    }
    if (tid == 0) {
        float m = sm.red_a[p][0], s = sm.red_b[p][0];
        for (int w = 1; w < kBlock / 64; ++w) lse_merge_finite(m, s, sm.red_a[p][w], sm.red_b[p][w]);
        uint64_t* part = (uint64_t*)(a.ws + a.L.part) + (size_t)row_id * a.L.nseg;
        st_dev(part + seg, ep | __float_as_uint(s));
    }
}

// ---------------------------------------------------------------- race search

__device__ __forceinline__ float current_threshold(Shared& sm) {
    return ordered_value(__hip_atomic_load(&sm.best_key, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP)) +
           kMargin;
}

__device__ __forceinline__ void push_node(Node* list, int* count, int cap, uint32_t id, float m, uint32_t p) {
    const int i = atomicAdd(count, 1);
    if (i < cap) list[i] = Node{id, m, p};
}

__device__ __forceinline__ void push_candidate(Shared& sm, const RaceArgs& a, int v, int j, float s, float x) {
    const int i = atomicAdd(&sm.n_cand, 1);
    if (i < kCandCap) {
        sm.cand_v[i] = v;
        sm.cand_j[i] = j;
        sm.cand_s[i] = s;
        sm.cand_x[i] = x;
    } else {
        set_error(a, kErrCand);
    }
}

// Keep only candidates within the margin of the current best (thread 0, between barriers).
__device__ __forceinline__ void compact_candidates(Shared& sm) {
    if (sm.n_cand <= kCandCap / 2) return;
    const float lim = ordered_value(sm.best_key) + kMargin;
    const int nc = min(sm.n_cand, kCandCap);
    int o = 0;
    for (int i = 0; i < nc; ++i)
        if (sm.cand_s[i] <= lim) {
            sm.cand_v[o] = sm.cand_v[i];
            sm.cand_j[o] = sm.cand_j[i];
            sm.cand_s[o] = sm.cand_s[i];
            sm.cand_x[o] = sm.cand_x[i];
            ++o;
        }
    sm.n_cand = o;
}

// Scores of the tokens of mask (bit t: token base4 + t) of one 4-token half, given
// the chunk's minimum (mc, pc) and the half's Philox words; INFINITY elsewhere and
// where the token cannot beat thr.
template <int LAYOUT>
__device__ __forceinline__ void half_scores(const Row& r, uint32_t base4, uint32_t mask, const float (&x)[4], float mc,
                                            uint32_t pc, const Words& w, float thr, float (&sc)[4]) {
    const uint32_t ws[4] = {w.w0, w.w1, w.w2, w.w3};
    const float lnmc = LAYOUT == 0 ? ln_f32(mc) : 0.f;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        sc[t] = INFINITY;
        if (!((mask >> t) & 1u)) continue;
        const uint32_t v = base4 + (uint32_t)t;
        if constexpr (LAYOUT == 0) {
            if (v == pc)
                sc[t] = lnmc - scaled(r, x[t]);
            else if (lnmc - scaled(r, x[t]) <= thr)
                sc[t] = ln_f32(mc + exp1_f32(ws[t])) - scaled(r, x[t]);
        } else {
            sc[t] = ln_f32(exp1_f32(ws[t])) - scaled(r, x[t]);
        }
    }
}

// Lower the best score to the half's smallest score.
__device__ __forceinline__ void offer_best(Shared& sm, const float (&sc)[4]) {
    const float mn = fminf(fminf(sc[0], sc[1]), fminf(sc[2], sc[3]));
    if (mn < INFINITY) atomicMin(&sm.best_key, ordered_key(mn));
}

// List the half's scores within the margin of the best as candidates.  Callers
// offer every half of the round first and separate the two steps by a barrier, so
// that only near-ties of the best are listed.
__device__ __forceinline__ void list_near(Shared& sm, const RaceArgs& a, uint32_t base4, uint32_t slot,
                                          const float (&sc)[4], const float (&x)[4]) {
    const float thr = current_threshold(sm);
#pragma unroll
    for (int t = 0; t < 4; ++t)
        if (sc[t] <= thr) push_candidate(sm, a, (int)(base4 + (uint32_t)t), (int)slot, sc[t], x[t]);
}

// Evaluate listed group entries [first, first + n): 16 lanes hold the 16 chunks of
// one entry (8 tokens each); each row takes kRowEntries entries, whose loads are
// issued together.  Only a few chunks of a surviving group hold a token that can
// still win against the group minimum (chunk and token minima are never below
// it), so the work is listed rather than done by each chunk's lane (a wave runs
// every branch any of its lanes takes): the 4-token halves that need token words
// go to an LDS list and are scored one per thread, each drawing its chunk's
// minimum too when the chunk does not hold the group's (two independent Philox
// calls).  Halves beyond the list's capacity are done by their chunk's lane.
// Raw logits of this lane's chunk of the entries of the pass starting at `first`
// (list end `end`; nothing is loaded past it).  Words past V are never used.
template <bool BF16, bool VEC>
__device__ __forceinline__ void load_pass(const RaceArgs& a, const Row& r, const Shared& sm, int first, int end,
                                          Unit<BF16, VEC> (&ux)[kRowEntries]) {
    const int c = threadIdx.x & 15, row = threadIdx.x >> 4;
#pragma unroll
    for (int q = 0; q < kRowEntries; ++q) {
        const int e = first + row * kRowEntries + q;
        if (e < end) {
            const uint32_t g = sm.l2[e].id & 0xFFFFFu;
            load_unit<BF16, VEC, false>(r.ptr, a.V, (int)(g * kGroupTokens + (uint32_t)c * 8u), ux[q]);
        }
    }
}

// The scored half a thread holds at the end of an evaluation pass (its logits stay
// in the half's list entry).
struct HalfOut {
    float sc[4];
    uint32_t base4, slot;
    bool valid;
};

template <bool BF16, bool VEC, int LAYOUT>
__device__ __forceinline__ void eval_groups(const RaceArgs& a, const Row& r, Shared& sm, const float* gm, int first,
                                            int n, int end, int par, uint32_t k0, uint32_t k1, HalfOut& ho,
                                            uint32_t& ovf, Unit<BF16, VEC> (&ux)[kRowEntries]) {
    const int tid = threadIdx.x, lane = tid & 63;
    const int c = tid & 15;
    const int row = tid >> 4;  // 16 rows of 16 lanes
    const uint32_t V = (uint32_t)a.V;
    constexpr uint32_t kDomain = LAYOUT == 0 ? kDomainTree : kDomainFlat;
    // this pass's logits were loaded into ux by the caller or the previous pass
    float x[kRowEntries][8];
    Node nd[kRowEntries];
    bool act[kRowEntries];
#pragma unroll
    for (int q = 0; q < kRowEntries; ++q) {
        const int e = first + row * kRowEntries + q;
        act[q] = e < first + n;
        nd[q] = act[q] ? sm.l2[e] : Node{0u, 0.f, 0u};
        unpack_unit<BF16, VEC>(ux[q], x[q]);
    }
    // What each chunk needs: its own draw (unless it holds the group minimum) and
    // the words of each half with a token that can still win.
    const float thr0 = current_threshold(sm);
    uint32_t hm[kRowEntries][2];
    bool cj[kRowEntries];
    int nh = 0;
#pragma unroll
    for (int q = 0; q < kRowEntries; ++q) {
        const uint32_t g = nd[q].id & 0xFFFFFu;
        const uint32_t base = g * kGroupTokens + (uint32_t)c * 8u;
        const float lnm = LAYOUT == 0 ? ln_f32(nd[q].m) : kLnClockFloor;
        hm[q][0] = hm[q][1] = 0u;
        cj[q] = false;
        if (act[q] && lnm - scaled(r, gm[g]) <= thr0) {
            // a token can reach thr0 only if lnm - (x - shift) / T <= thr0, i.e.
            // x - shift >= (lnm - thr0) T; the cut is lowered by kCutSlack, far more
            // than the rounding of either form, so the listed tokens include every
            // such token (compared in the shifted frame: no rounding of shift + cut)
            const float xc = (lnm - thr0 - kCutSlack) * r.T;
            uint32_t m8 = 0u;
#pragma unroll
            for (int i = 0; i < 8; ++i) m8 |= (uint32_t)(x[q][i] - r.shift >= xc) << i;
            const int nv = (int)V - (int)base;  // tokens of this chunk inside the row
            if (nv < 8) m8 &= nv > 0 ? (1u << nv) - 1u : 0u;
            hm[q][0] = m8 & 15u;
            hm[q][1] = m8 >> 4;
            if (LAYOUT == 0 && m8) {
                const uint32_t ce = node_end(kShift1, g * 16u + (uint32_t)c, V);
                cj[q] = !(nd[q].p >= base && nd[q].p < ce);
            }
        }
        nh += (int)(hm[q][0] != 0u) + (int)(hm[q][1] != 0u);
    }
    // list positions: wave prefix sum of the halves, one atomic per wave
    const uint32_t mine = (uint32_t)nh;
    const uint32_t incl = wave_incl_sum(mine);
    const uint32_t wtot = (uint32_t)__builtin_amdgcn_readlane((int)incl, 63);
    uint32_t wbase = 0u;
    if (lane == 0 && wtot != 0u) wbase = atomicAdd(&sm.n_ev[par], wtot);
    const uint32_t mb = (uint32_t)__builtin_amdgcn_readlane((int)wbase, 0) + incl - mine;
    int jh = (int)mb;
    ovf = 0u;  // halves beyond the list (bit 8q + 4h + t: token t of half h of entry q)
#pragma unroll
    for (int q = 0; q < kRowEntries; ++q) {
        const int le = row * kRowEntries + q;
        const int cref = cj[q] ? 0 : -1;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            if (hm[q][h]) {
                if (jh < kHalfCap) {
                    Half& hf = sm.half[jh];
                    hf.desc = ((uint32_t)le << 9) | ((uint32_t)c << 5) | ((uint32_t)h << 4) | hm[q][h];
                    hf.cref = cref;
                    hf.x[0] = x[q][4 * h];
                    hf.x[1] = x[q][4 * h + 1];
                    hf.x[2] = x[q][4 * h + 2];
                    hf.x[3] = x[q][4 * h + 3];
                } else {
                    ovf |= hm[q][h] << (8 * q + 4 * h);
                }
                ++jh;
            }
        }
    }
    // the next pass's logits, in flight while this pass draws and scores
    load_pass<BF16, VEC>(a, r, sm, first + kPassGroups, end, ux);
    __syncthreads();
    // the other parity's counts were read in the previous pass: clear them for the next
    if (tid == 0) sm.n_ev[par ^ 1] = 0u;
    // halves, one per thread (at most one: kHalfCap == kBlock): scores, and the best
    // lowered to each half's smallest; the caller lists near-ties after a barrier
    static_assert(kHalfCap == kBlock, "one listed half per thread");
    {
        const int nj = min((int)sm.n_ev[par], kHalfCap);
        const float thr = current_threshold(sm);
#pragma unroll
        for (int t = 0; t < 4; ++t) ho.sc[t] = INFINITY;
        ho.base4 = ho.slot = 0u;
        ho.valid = tid < nj;
        if (ho.valid) {
            const Half hf = sm.half[tid];
            const Node pn = sm.l2[first + (int)(hf.desc >> 9)];
            ho.slot = pn.id >> 20;
            const uint32_t g = pn.id & 0xFFFFFu;
            const uint32_t chunk = g * 16u + ((hf.desc >> 5) & 15u), h = (hf.desc >> 4) & 1u;
            ho.base4 = chunk * 8u + 4u * h;
            float mc = pn.m;
            uint32_t pc = pn.p;
            if (LAYOUT == 0 && hf.cref >= 0) {
                // the chunk's own minimum (its draw is independent of the half's words,
                // so the two Philox calls overlap)
                const uint32_t ce = node_end(kShift1, chunk, V);
                const Words wc = philox(chunk, ho.slot, 1u, kDomainTree, k0, k1);
                mc = pn.m + div_n(exp1_f32(wc.w0), ce - chunk * 8u);
                pc = chunk * 8u + uniform_position(wc.w1, wc.w2, ce - chunk * 8u);
            }
            const Words w = LAYOUT == 0 ? philox(chunk, ho.slot, 8u + h, kDomainTree, k0, k1)
                                        : philox(ho.base4 >> 2, ho.slot, 0u, kDomainFlat, k0, k1);
            half_scores<LAYOUT>(r, ho.base4, hf.desc & 15u, hf.x, mc, pc, w, thr, ho.sc);
            offer_best(sm, ho.sc);
        }
    }
}

// Halves an evaluation pass could not list (more than kHalfCap): each is scored by
// its chunk's lane (logits read again), one (entry, half) combination at a time,
// with the same offer / barrier / list steps.  Called by every thread.
template <bool BF16, int LAYOUT>
__device__ __forceinline__ void eval_overflow(const RaceArgs& a, const Row& r, Shared& sm, int first, uint32_t ovf,
                                              uint32_t k0, uint32_t k1) {
    const int tid = threadIdx.x, c = tid & 15, row = tid >> 4;
    const uint32_t V = (uint32_t)a.V;
    // (rare: one copy of the code, not unrolled)
#pragma unroll 1
    for (int q = 0; q < kRowEntries; ++q) {
#pragma unroll 1
        for (int h = 0; h < 2; ++h) {
            const uint32_t mask = (ovf >> (8 * q + 4 * h)) & 15u;
            float sc[4] = {INFINITY, INFINITY, INFINITY, INFINITY}, xs[4] = {0.f, 0.f, 0.f, 0.f};
            uint32_t base4 = 0u, slot = 0u;
            if (mask != 0u) {
                const Node pn = sm.l2[first + row * kRowEntries + q];
                slot = pn.id >> 20;
                const uint32_t g = pn.id & 0xFFFFFu;
                const uint32_t chunk = g * 16u + (uint32_t)c;
                base4 = chunk * 8u + 4u * (uint32_t)h;
                float mc = pn.m;
                uint32_t pc = pn.p;
                const uint32_t ce = node_end(kShift1, chunk, V);
                if (LAYOUT == 0 && !(pn.p >= chunk * 8u && pn.p < ce)) {
                    const Words wc = philox(chunk, slot, 1u, kDomainTree, k0, k1);
                    mc = pn.m + div_n(exp1_f32(wc.w0), ce - chunk * 8u);
                    pc = chunk * 8u + uniform_position(wc.w1, wc.w2, ce - chunk * 8u);
                }
                const Words w = LAYOUT == 0 ? philox(chunk, slot, 8u + (uint32_t)h, kDomainTree, k0, k1)
                                            : philox(base4 >> 2, slot, 0u, kDomainFlat, k0, k1);
#pragma unroll
                for (int t = 0; t < 4; ++t)
                    xs[t] = (mask >> t) & 1u ? load_logit<BF16>(r.ptr, (int)(base4 + (uint32_t)t)) : -INFINITY;
                half_scores<LAYOUT>(r, base4, mask, xs, mc, pc, w, current_threshold(sm), sc);
                offer_best(sm, sc);
            }
            __syncthreads();
            if (mask != 0u) list_near(sm, a, base4, slot, sc, xs);
            __syncthreads();
        }
    }
}

// Reorder the first n entries of the group list by their bounds (ln of the group
// minimum minus the scaled group maximum), counting-sorted into kBuckets buckets
// between the smallest bound and the threshold; entries above the threshold are
// dropped.  Evaluating the most promising groups first lowers the threshold
// early, and a pass whose first entry's bucket lies above the threshold ends the
// evaluation (later buckets hold larger bounds).  Returns the kept count.  The
// sort stages the list in half[], which is free between evaluation passes.
// Called by every thread.
template <int LAYOUT>
__device__ __forceinline__ int order_groups(const Row& r, Shared& sm, const float* gm, int n) {
    static_assert(kL2Cap <= 2 * kBlock, "two entries per thread");
    const int tid = threadIdx.x, lane = tid & 63;
    const float thr = current_threshold(sm);
    Node nd[2];
    float b[2];
    float wmin = INFINITY;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int e = tid + i * kBlock;
        nd[i] = e < n ? sm.l2[e] : Node{0u, 0.f, 0u};
        const float lnm = LAYOUT == 0 ? ln_f32(nd[i].m) : kLnClockFloor;
        b[i] = e < n ? lnm - scaled(r, gm[nd[i].id & 0xFFFFFu]) : INFINITY;
        if (b[i] <= thr) wmin = fminf(wmin, b[i]);
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) wmin = fminf(wmin, __shfl_xor(wmin, off));
    if (lane == 0) sm.ord_wmin[tid >> 6] = wmin;
    if (tid < kBuckets) {
        sm.ord_hist[tid] = 0;
        sm.ord_bmin[tid] = ordered_key(INFINITY);
    }
    __syncthreads();
    float bmin = sm.ord_wmin[0];
#pragma unroll
    for (int w = 1; w < kBlock / 64; ++w) bmin = fminf(bmin, sm.ord_wmin[w]);
    // bucket = floor((b - bmin) * scale), non-decreasing in b
    const float scale = thr > bmin ? (float)kBuckets / (thr - bmin) : 0.f;
    int k[2], rank[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        k[i] = -1;
        rank[i] = 0;
        if (b[i] <= thr) {
            k[i] = min(kBuckets - 1, (int)((b[i] - bmin) * scale));
            rank[i] = atomicAdd(&sm.ord_hist[k[i]], 1);
            atomicMin(&sm.ord_bmin[k[i]], ordered_key(b[i]));
        }
    }
    __syncthreads();
    // bucket starts: a prefix sum over the kBuckets counts in every wave
    const int h = lane < kBuckets ? sm.ord_hist[lane] : 0;
    int incl = h;
#pragma unroll
    for (int off = 1; off < kBuckets; off <<= 1) {
        const int o = __shfl_up(incl, off);
        if (lane >= off) incl += o;
    }
    const int excl = incl - h;
    const int kept = __shfl(incl, kBuckets - 1);
    Node* tmp = reinterpret_cast<Node*>(sm.half);
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int start = __shfl(excl, max(k[i], 0));
        if (k[i] >= 0) {
            const int dst = start + rank[i];
            tmp[dst] = nd[i];
            if (dst % kPassGroups == 0) sm.ord_pass[dst / kPassGroups] = k[i];
        }
    }
    __syncthreads();
    for (int e = tid; e < kept; e += kBlock) sm.l2[e] = tmp[e];
    __syncthreads();
    return kept;
}

// Evaluate and empty the group list.  Callers read the list count after a barrier
// and before any push of the current pass.
template <bool BF16, bool VEC, int LAYOUT>
__device__ __forceinline__ void flush_groups(const RaceArgs& a, const Row& r, Shared& sm, const float* gm, uint32_t k0,
                                             uint32_t k1) {
    int n = min(sm.n_l2, kL2Cap);
    const bool ordered = n > kPassGroups;
    if (ordered) n = order_groups<LAYOUT>(r, sm, gm, n);
    int par = 0;
    Unit<BF16, VEC> ux[kRowEntries];
    load_pass<BF16, VEC>(a, r, sm, 0, n, ux);
    for (int first = 0; first < n; first += kPassGroups, par ^= 1) {
        // every later entry's bound is at least its bucket's smallest (the threshold
        // and the buckets are read after the previous pass's last barrier)
        if (ordered && first > 0 && ordered_value(sm.ord_bmin[sm.ord_pass[first / kPassGroups]]) > current_threshold(sm))
            break;
        HalfOut ho;
        uint32_t ovf;
        eval_groups<BF16, VEC, LAYOUT>(a, r, sm, gm, first, min(n - first, kPassGroups), n, par, k0, k1, ho, ovf, ux);
        __syncthreads();
        // every half of the pass has lowered the best: list the near-ties
        if (ho.valid) list_near(sm, a, ho.base4, ho.slot, ho.sc, sm.half[threadIdx.x].x);
        if (sm.n_ev[par] > (uint32_t)kHalfCap) eval_overflow<BF16, LAYOUT>(a, r, sm, first, ovf, k0, k1);
        __syncthreads();
        // (the next pass touches the candidates only after two more barriers)
        if (threadIdx.x == 0) compact_candidates(sm);
    }
    if (threadIdx.x == 0) {
        sm.n_l2 = 0;
        sm.n_ev[0] = sm.n_ev[1] = 0u;
    }
    __syncthreads();
}

// Expand listed level-3 nodes into groups (tree clocks), evaluating the groups as
// the list fills.  A draw-free prefilter (group maximum against the node's
// minimum) first compacts the (node, group) items that can still win into a work
// list, so that the draws run on full wavefronts.  One loop with a single
// evaluation call site: it refills the work list when it is used up, evaluates the
// group list when it may overflow or at the end, and draws kBlock items per step.
template <bool BF16, bool VEC>
__device__ __forceinline__ void flush_l3(const RaceArgs& a, const Row& r, Shared& sm, const float* gm, uint32_t k0, uint32_t k1) {
    const int tid = threadIdx.x;
    const int n = min(sm.n_l3, kL3Cap) * 16;
    const uint32_t V = (uint32_t)a.V;
    const int ng = a.L.ng;
    int base = 0, nw = 0, wb = 0;  // next prefilter item; work list size; next work item
    for (;;) {
        // (uniform: nw is read by every thread after a barrier; a list found empty
        // is 0 when thread 0 clears it again)
        while (wb >= nw && base < n) {
            if (tid == 0) sm.n_work = 0;
            __syncthreads();
            const float thr = current_threshold(sm);
            for (int e = base + tid; e < min(n, base + kWorkCap); e += kBlock) {
                const Node pa = sm.l3[e >> 4];
                const uint32_t g = (pa.id & 0xFFFFFu) * 16u + (uint32_t)(e & 15);
                if ((int)g < ng && ln_f32(pa.m) - scaled(r, gm[g]) <= thr) sm.work[atomicAdd(&sm.n_work, 1)] = e;
            }
            __syncthreads();
            nw = sm.n_work;
            wb = 0;
            base += kWorkCap;
        }
        const bool done = wb >= nw;
        // The count is read by every thread before any thread of this step pushes.
        const bool flush = done ? sm.n_l2 > 0 : sm.n_l2 > kL2Cap - kBlock;
        __syncthreads();
        if (flush) flush_groups<BF16, VEC, 0>(a, r, sm, gm, k0, k1);
        if (done) break;
        const int i = wb + tid;
        if (i < nw) {
            const int e = sm.work[i];
            const Node pa = sm.l3[e >> 4];
            const uint32_t g = (pa.id & 0xFFFFFu) * 16u + (uint32_t)(e & 15);
            const float thr = current_threshold(sm);
            if (ln_f32(pa.m) - scaled(r, gm[g]) <= thr) {
                const uint32_t slot = pa.id >> 20;
                float m;
                uint32_t p;
                child_min_f32(pa.m, pa.p, 2, g, g << kShift2, node_end(kShift2, g, V), slot, k0, k1, m, p);
                if (ln_f32(m) - scaled(r, gm[g]) <= thr) push_node(sm.l2, &sm.n_l2, kL2Cap, (slot << 20) | g, m, p);
            }
        }
        wb += kBlock;
        __syncthreads();
    }
    if (tid == 0) sm.n_l3 = 0;
    __syncthreads();
}

// Lexicographic minimum of (score, token, slot).
__device__ __forceinline__ bool lex_less(double s, int v, int j, double s2, int v2, int j2) {
    return s < s2 || (s == s2 && (v < v2 || (v == v2 && j < j2)));
}

__device__ __forceinline__ int path_shift(int l) {
    return l == 1 ? kShift4 : l == 2 ? kShift3 : l == 3 ? kShift2 : kShift1;
}

// Counter words (c0, c2) of path node l of token v (tree clocks): 0 = root, 1..4 =
// the token's level-4..1 ancestors, 5 = the token's own word block.  The counter
// is selected per lane, so lanes of one token draw their nodes in a single call.
__device__ __forceinline__ uint32_t path_c0(int l, uint32_t v) { return l == 0 ? 0u : l == 5 ? v >> 3 : v >> path_shift(l); }
__device__ __forceinline__ uint32_t path_c2(int l, uint32_t v) {
    return l == 0 ? 5u : l == 5 ? 8u + ((v >> 2) & 1u) : (uint32_t)(5 - l);
}
__device__ __forceinline__ Words path_draw(int l, uint32_t v, uint32_t slot, uint32_t k0, uint32_t k1) {
    return philox(path_c0(l, v), slot, path_c2(l, v), kDomainTree, k0, k1);
}

__device__ __forceinline__ uint32_t pick_word(uint32_t a0, uint32_t a1, uint32_t a2, uint32_t a3, uint32_t i) {
    return i == 0 ? a0 : i == 1 ? a1 : i == 2 ? a2 : a3;
}

template <bool BF16, bool VEC, int LAYOUT>
__device__ __forceinline__ void race(const RaceArgs& a, const Row& r, Shared& sm, const float* gm, uint32_t k0, uint32_t k1) {
    // (lists, candidates and the best score were reset by the caller)
    const int tid = threadIdx.x;
    const uint32_t V = (uint32_t)a.V;
    const int ng = a.L.ng;
    const int ns = r.nslots;
    const int n4 = (int)((V + (1u << kShift4) - 1) >> kShift4);
    // Pass A: the seed tokens (each the largest logit of its group) in every slot --
    // tree clocks: 8 lanes per (token, slot), lane l < 6 drawing path node l -- and,
    // for tree clocks, the minimum of every (slot, level-4 node): lanes 6 and 7 of the
    // seed lanes of slot j take its first 2 kInit level-4 nodes (with the root drawn
    // by lane 0), lanes past the seed lanes the rest, one item per lane.
    const int nseed = kInit;
    const int seed_lanes = nseed * ns * 8;
    const int n4x = max(0, n4 - 2 * nseed);  // level-4 nodes per slot past the seed lanes
    const int nA = seed_lanes + (LAYOUT == 0 ? ns * n4x : 0);
    for (int e0 = 0; e0 < nA; e0 += kBlock) {
        const int e = e0 + tid;
        if (e < seed_lanes) {  // whole 8-lane groups: the shuffles stay within active lanes
            const int pair = e >> 3, l = e & 7;
            static_assert(kInit == 8, "seed index = low 3 bits of the 8-lane group index");
            const int w = pair & 7, j = pair >> 3;  // seed w, slot j
            const int tv = sm.seed_tok[w];
            const int g = tv >= 0 ? tv >> 7 : -1;
            const uint32_t slot = (uint32_t)(r.slot0 + j);
            const uint32_t av = (uint32_t)max(tv, 0);
            const float xa = g >= 0 ? gm[g] : -INFINITY;
            if constexpr (LAYOUT == 0) {
                // lane l turns node l's draw into (minimum increment, position): root
                // E'/V, level-4..1 node E'/size at a uniform position in it, token E'
                float val = 0.f;
                uint32_t pos = 0u;
                const uint32_t i4 = (uint32_t)(2 * w + (l - 6));  // level-4 node of lanes 6 and 7
                const bool l4 = l >= 6 && (int)i4 < n4;
                if (l < 6 || l4) {
                    const Words wd = philox(l4 ? i4 : path_c0(l, av), slot, l4 ? 4u : path_c2(l, av), kDomainTree, k0, k1);
                    const int sh = l4 ? kShift4 : path_shift(l);
                    const uint32_t node = l4 ? i4 : av >> sh;
                    const uint32_t cs = (l == 0 || l == 5) ? 0u : node << sh;
                    const uint32_t n = l == 0 ? V : l == 5 ? 1u : node_end(sh, node, V) - cs;
                    val = div_n(exp1_f32(l == 5 ? pick_word(wd.w0, wd.w1, wd.w2, wd.w3, av & 3u) : wd.w0), n);
                    pos = cs + uniform_position(wd.w1, wd.w2, n);
                }
                const int base = tid & ~7;
                float m = __shfl(val, base);
                uint32_t p = (uint32_t)__shfl((int)pos, base);
                if (l4) {
                    // the root (lane 0) or this node holds the level-4 node's minimum
                    const uint32_t cs = i4 << kShift4, ce = node_end(kShift4, i4, V);
                    const bool hold = p >= cs && p < ce;
                    level4_list(gm, ng)[j * n4 + (int)i4] =
                        Node{(slot << 20) | i4, hold ? m : m + val, hold ? p : pos};
                }
#pragma unroll
                for (int q = 1; q <= 4; ++q) {
                    const float vq = __shfl(val, base + q);
                    const uint32_t pq = (uint32_t)__shfl((int)pos, base + q);
                    const int sh = path_shift(q);
                    const uint32_t i = av >> sh, cs = i << sh, ce = node_end(sh, i, V);
                    if (!(p >= cs && p < ce)) {
                        m = m + vq;
                        p = pq;
                    }
                }
                const float v5 = __shfl(val, base + 5);
                const float E = (av == p) ? m : m + v5;
                if (l == 0 && g >= 0) {
                    const float sc = ln_f32(E) - scaled(r, xa);
                    if (sc < INFINITY) {
                        atomicMin(&sm.best_key, ordered_key(sc));
                        push_candidate(sm, a, (int)av, (int)slot, sc, xa);
                    }
                }
            } else {
                if (l == 0 && g >= 0) {
                    const Words wd = philox(av >> 2, slot, 0u, kDomainFlat, k0, k1);
                    const float sc = ln_f32(exp1_f32(word_at(wd, av & 3u))) - scaled(r, xa);
                    if (sc < INFINITY) {
                        atomicMin(&sm.best_key, ordered_key(sc));
                        push_candidate(sm, a, (int)av, (int)slot, sc, xa);
                    }
                }
            }
        } else if (LAYOUT == 0 && e < nA) {
            // level-4 node i4 of slot j past the seed lanes: root and node draws
            // issued together
            const int it = e - seed_lanes, j = it / n4x;
            const uint32_t i4 = (uint32_t)(2 * nseed + it % n4x);
            const uint32_t slot = (uint32_t)(r.slot0 + j);
            const Words wr = philox(0u, slot, 5u, kDomainTree, k0, k1);
            const Words w4 = philox(i4, slot, 4u, kDomainTree, k0, k1);
            const float rm = div_n(exp1_f32(wr.w0), V);
            const uint32_t rp = uniform_position(wr.w1, wr.w2, V);
            const uint32_t cs = i4 << kShift4, n = node_end(kShift4, i4, V) - cs;
            const bool hold = rp >= cs && rp < cs + n;
            level4_list(gm, ng)[j * n4 + (int)i4] = Node{(slot << 20) | i4, hold ? rm : rm + div_n(exp1_f32(w4.w0), n),
                             hold ? rp : cs + uniform_position(w4.w1, w4.w2, n)};
        }
    }
    __syncthreads();

    if constexpr (LAYOUT == 0) {
        // Pass B: level-3 children of the level-4 nodes that can still win.
        const int nB = ns * n4 * 16;
        const int n3 = (ng + 15) / 16;
        for (int base = 0;; base += kBlock) {
            const bool done = base >= nB;  // one call site of flush_l3 (see flush_l3)
            const bool flush = done || sm.n_l3 > kL3Cap - kBlock;
            __syncthreads();
            if (flush) flush_l3<BF16, VEC>(a, r, sm, gm, k0, k1);
            if (done) break;
            const int e = base + tid;
            if (e < nB) {
                const Node pa = level4_list(gm, ng)[e >> 4];
                const uint32_t i4 = pa.id & 0xFFFFFu;
                const uint32_t i3 = i4 * 16u + (uint32_t)(e & 15);
                const float thr = current_threshold(sm);
                const float lnp = ln_f32(pa.m);
                if ((int)i3 < n3 && lnp - scaled(r, sm.m4[i4]) <= thr && lnp - scaled(r, sm.m3[i3]) <= thr) {
                    const uint32_t slot = pa.id >> 20;
                    float m;
                    uint32_t p;
                    child_min_f32(pa.m, pa.p, 3, i3, i3 << kShift3, node_end(kShift3, i3, V), slot, k0, k1, m, p);
                    if (ln_f32(m) - scaled(r, sm.m3[i3]) <= thr) push_node(sm.l3, &sm.n_l3, kL3Cap, (slot << 20) | i3, m, p);
                }
            }
            __syncthreads();
        }
    } else {
        // flat clocks: every (group, slot) whose floor bound can win.
        const int tot = ng * ns;
        for (int base = 0;; base += kBlock) {
            const bool done = base >= tot;  // one call site of flush_groups
            const bool flush = done || sm.n_l2 > kL2Cap - kBlock;
            __syncthreads();
            if (flush) flush_groups<BF16, VEC, 1>(a, r, sm, gm, k0, k1);
            if (done) break;
            const int e = base + tid;
            if (e < tot) {
                const int g = e / ns;
                const uint32_t slot = (uint32_t)(r.slot0 + e % ns);
                if (kLnClockFloor - scaled(r, gm[g]) <= current_threshold(sm))
                    push_node(sm.l2, &sm.n_l2, kL2Cap, (slot << 20) | (uint32_t)g, 0.f, 0u);
            }
            __syncthreads();
        }
    }

    // decide: float64 scores of the candidates within the margin of the best; for
    // tree clocks 8 lanes per candidate draw its path nodes in parallel.
    const float best = ordered_value(sm.best_key);
    const int nc = min(sm.n_cand, kCandCap);
    {
        // A single candidate within the margin of the best is the winner: float32
        // scores err by far less than the margin, and every token that was not kept
        // scored above it.
        static_assert(kCandCap <= kBlock, "one candidate per thread");
        const bool in = tid < nc && sm.cand_s[tid] <= best + kMargin;
        if (in) {
            const int key = sm.cand_v[tid] * 32 + sm.cand_j[tid];  // token < 2^19, slot < 32
            atomicMin(&sm.key_min, key);
            atomicMax(&sm.key_max, key);
            sm.win_token = sm.cand_v[tid];
            sm.win_slot = sm.cand_j[tid];
        }
        __syncthreads();
        if (sm.key_min == sm.key_max) return;  // one (token, slot), possibly listed twice
        __syncthreads();
    }
    double bs = INFINITY;
    int bv = 0x7FFFFFFF, bj = 0x7FFFFFFF;
    for (int e0 = 0; e0 < nc * 8; e0 += kBlock) {
        const int e = e0 + tid;
        const int ci = e >> 3, l = e & 7;
        const bool valid = ci < nc && sm.cand_s[ci] <= best + kMargin;
        const int v = valid ? sm.cand_v[ci] : 0, j = valid ? sm.cand_j[ci] : 0;
        double E = 0.0;
        if constexpr (LAYOUT == 0) {
            Words wd = Words{0u, 0u, 0u, 0u};
            if (valid && l < 6) wd = path_draw(l, (uint32_t)v, (uint32_t)j, k0, k1);
            double m = 0.0;
            uint32_t p = 0u;
#pragma unroll
            for (int q = 0; q < 6; ++q) {
                const int src = (tid & ~7) + q;
                const uint32_t a0 = (uint32_t)__shfl((int)wd.w0, src);
                const uint32_t a1 = (uint32_t)__shfl((int)wd.w1, src);
                const uint32_t a2 = (uint32_t)__shfl((int)wd.w2, src);
                const uint32_t a3 = (uint32_t)__shfl((int)wd.w3, src);
                if (l != 0 || !valid) continue;
                if (q == 0) {
                    m = exp1_f64(a0) / (double)V;
                    p = uniform_position(a1, a2, V);
                } else if (q <= 4) {
                    const int sh = path_shift(q);
                    const uint32_t i = (uint32_t)v >> sh, cs = i << sh, ce = node_end(sh, i, V);
                    if (!(p >= cs && p < ce)) {
                        m = m + exp1_f64(a0) / (double)(ce - cs);
                        p = cs + uniform_position(a1, a2, ce - cs);
                    }
                } else {
                    E = ((uint32_t)v == p) ? m : m + exp1_f64(pick_word(a0, a1, a2, a3, (uint32_t)v & 3u));
                }
            }
        } else {
            if (l == 0 && valid) E = flat_clock_f64((uint32_t)j, (uint32_t)v, k0, k1);
        }
        if (l == 0 && valid) {
            const double s = log(E) - (double)sm.cand_x[ci] / (double)r.T;
            if (lex_less(s, v, j, bs, bv, bj)) {
                bs = s;
                bv = v;
                bj = j;
            }
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

__device__ __forceinline__ int walk_draft(const RaceArgs& a, int b, int k, int s, uint32_t ep) {
    if (a.s_count > 0 && s >= a.s_begin) return wait_token(a, draft_row_id(a, b, k, s), ep);
    return a.draft_tokens[((size_t)b * a.K + k) * a.gamma + s];
}

// Realised-path walk of sequence b; every token it reads carries this call's epoch.
// Called by every thread: the tokens the walk may read are fetched in parallel
// first (into the candidate arrays, free once the race is decided); thread 0 walks.
__device__ __forceinline__ void walk(const RaceArgs& a, Shared& sm, int b, uint32_t ep) {
    const int K = a.K, G = a.gamma, tid = threadIdx.x;
    const int ntp = a.target_rows == 1 ? 1 : K;
    const int nt = ntp * (G + 1), n = nt + K * G;
    const bool staged = n <= kCandCap;
    if (staged) {
        for (int e = tid; e < n; e += kBlock)
            sm.cand_v[e] = e < nt ? wait_token(a, target_row_id(a, b, e / (G + 1), e % (G + 1)), ep)
                                  : walk_draft(a, b, (e - nt) / G, (e - nt) % G, ep);
        __syncthreads();
    }
    if (tid != 0) return;
    auto target = [&](int k, int s) {
        return staged ? sm.cand_v[(ntp == 1 ? 0 : k) * (G + 1) + s] : wait_token(a, target_row_id(a, b, k, s), ep);
    };
    auto draft = [&](int k, int s) { return staged ? sm.cand_v[nt + k * G + s] : walk_draft(a, b, k, s, ep); };
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
            if (((act >> k) & 1u) && draft(k, s) == y) na |= 1u << k;
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

// ---------------------------------------------------------------- row finisher

// Token at path depth d of this row's context (prefix excluded).
__device__ __forceinline__ int path_token(const RaceArgs& a, const Row& r, int d, uint32_t ep) {
    if (r.kind == 1 && a.target_rows == 1) return wait_token(a, target_row_id(a, r.b, 0, d), ep);
    if (a.s_count > 0 && d >= a.s_begin) return wait_token(a, draft_row_id(a, r.b, r.k, d), ep);
    return a.draft_tokens[((size_t)r.b * a.K + r.k) * a.gamma + d];
}

// Row whose race publishes this row's context key (-1: the key is folded here, all
// its tokens being known before the call).  The key of depth s of a path is
// finished by the race at depth s - 1, which alone knows the newest token.
__device__ __forceinline__ int key_producer(const RaceArgs& a, const Row& r) {
    if (a.m == 0 || r.s == 0) return -1;
    if (r.kind == 1 && a.target_rows == 1) return target_row_id(a, r.b, 0, r.s - 1);
    if (a.s_count > 0 && r.s - 1 >= a.s_begin && r.s - 1 < a.s_begin + a.s_count)
        return draft_row_id(a, r.b, r.k, r.s - 1);
    return -1;
}

// Whether this row's race publishes the context key of the next depth of its path.
__device__ __forceinline__ bool key_consumer(const RaceArgs& a, const Row& r) {
    if (a.m == 0) return false;
    if (r.kind == 1) return a.target_rows == 1 && r.s + 1 <= a.gamma;
    return r.s + 1 < a.s_begin + a.s_count || (a.target_rows > 1 && r.s + 1 <= a.gamma);
}

template <bool BF16, bool VEC, int LAYOUT>
__device__ __forceinline__ void finish_row(const RaceArgs& a, const Row& r, Shared& sm, float* gm) {
    // The race is a latency chain (the next depth of this path waits for it) while
    // the other waves on the same SIMDs stream: raise this wave's issue priority,
    // the most for target rows, whose chain is one race longer than a draft path's
    // and ends the launch (102.4 vs 101.7 µs at V = 128256, K = 4, B = 64 against
    // one shared priority; drafts at the streamers' priority: 104 µs).
    if (r.kind == 1)
        __builtin_amdgcn_s_setprio(3);
    else
        __builtin_amdgcn_s_setprio(1);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int ng = a.L.ng;
    const int n3 = (ng + 15) / 16, n4 = (n3 + 15) / 16;
    const uint32_t ep = sm.epoch;
    const float c2 = r.invT * 1.4426950408889634f;

    // Context-key inputs known before the call (prompt tokens, position) are loaded
    // first, so their latency overlaps the gather.  Wave 3 lanes [0, m) take this
    // row's own window (when no race of this call publishes its key), lanes
    // [m, 2m - 1) the next depth's window without its newest token (when this race
    // publishes the next key); positions index prefix (m tokens) || path.
    const int prod = key_producer(a, r);
    const bool cons = key_consumer(a, r);
    int widx = -1, wtok = 0;
    int64_t wpos = 0;
    if (wave == 3) {
        if (lane < a.m && prod < 0)
            widx = r.s + lane;
        else if (lane >= a.m && lane < 2 * a.m - 1 && cons)
            widx = r.s + 1 + (lane - a.m);
        if (widx >= 0 && widx < a.m) wtok = a.prefix[(size_t)r.b * a.m + widx];
        wpos = a.start_pos[r.b];
    }

    // ---- gather the row's slots (group maxima, block maxima, segment top tokens):
    // a batch of loads in flight per thread, then a wait only for slots not yet
    // published.
    {
        const uint64_t* gslot = (const uint64_t*)(a.ws + a.L.gmax) + (size_t)r.row_id * ng;
        const uint64_t* m3slot = (const uint64_t*)(a.ws + a.L.m3) + (size_t)r.row_id * n3;
        const uint64_t* stop = (const uint64_t*)(a.ws + a.L.stop) + (size_t)r.row_id * a.L.nseg;
        const uint64_t* pslot = (const uint64_t*)(a.ws + a.L.part) + (size_t)r.row_id * a.L.nseg;
        const int ne = ng + n3 + 2 * a.L.nseg;
        for (int e0 = 0; e0 < ne; e0 += 4 * kBlock) {
            const uint64_t* src[4];
            uint64_t v[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int e = e0 + i * kBlock + tid;
                src[i] = e < ng                     ? gslot + e
                         : e < ng + n3                ? m3slot + (e - ng)
                         : e < ng + n3 + a.L.nseg     ? stop + (e - ng - n3)
                                                      : pslot + min(e - ng - n3 - a.L.nseg, a.L.nseg - 1);
                v[i] = e < ne ? ld_dev(src[i]) : 0;
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int e = e0 + i * kBlock + tid;
                if (e < ne) {
                    if ((uint32_t)(v[i] >> 32) != ep) v[i] = wait_slot(a, src[i], ep);
                    const uint32_t w = (uint32_t)v[i];
                    if (e < ng)
                        gm[e] = __uint_as_float(w);
                    else if (e < ng + n3)
                        sm.m3[e - ng] = __uint_as_float(w);
                    else if (e < ng + n3 + a.L.nseg)  // a group index of this row, or -1 (a value
                        sm.stop[e - ng - n3] = (int)w >= -1 && (int)w < ng ? (int)w : -1;  // left stale by a timed-out wait is dropped)
                    else
                        sm.part[e - ng - n3 - a.L.nseg] = __uint_as_float(w);
                }
            }
        }
    }
    __syncthreads();

    // ---- key-independent work: the race's seed tokens (the largest token of each
    // segment's top group, at most kInit of the largest groups), level-4 maxima,
    // LSE, row maximum.
    if (wave == 0) {
        float bv = -INFINITY;
        int bt = 0x7FFFFFFF;
        if (lane < a.L.nseg && sm.stop[lane] >= 0) {
            bt = sm.stop[lane];
            bv = gm[bt];
        }
        if (a.L.nseg <= kInit) {
            if (lane < kInit) sm.init_v[lane] = bv == -INFINITY ? -1 : bt;
        } else {
            for (int i = 0; i < kInit; ++i) {
                float mv = bv;
                int mt = bt;
#pragma unroll
                for (int off = 32; off > 0; off >>= 1) {
                    const float ov = __shfl_xor(mv, off);
                    const int ot = __shfl_xor(mt, off);
                    if (ov > mv || (ov == mv && ot < mt)) {
                        mv = ov;
                        mt = ot;
                    }
                }
                if (lane == 0) sm.init_v[i] = mv == -INFINITY ? -1 : mt;
                if (bt == mt) bv = -INFINITY;
            }
        }
    }
    __syncthreads();
    // Waves 0-1: the seed tokens, 16 lanes per seed group with 8 tokens each (the
    // group's lowest token holding its maximum); wave 2: level-4 maxima, LSE, row
    // maximum; wave 3: the context keys.  The four run side by side.
    if (wave < 2) {
        static_assert(kInit * 16 == 128, "one 16-lane row per seed group in waves 0-1");
        const int i = tid >> 4, sub = tid & 15;
        const int g = sm.init_v[i];
        int tk = 0x7FFFFFFF;
        if (g >= 0) {
            float x[8];
            const int base = g * kGroupTokens + sub * 8;
            load8<BF16, VEC>(r.ptr, a.V, base, x);
            const float gmax = gm[g];
#pragma unroll
            for (int t = 7; t >= 0; --t)
                if (base + t < a.V && x[t] == gmax) tk = base + t;
        }
#pragma unroll
        for (int off = 8; off > 0; off >>= 1) tk = min(tk, __shfl_xor(tk, off));
        if (sub == 0) sm.seed_tok[i] = g >= 0 && tk != 0x7FFFFFFF ? tk : -1;
    } else if (wave == 2) {
        if (lane < n4) {
            float mx = -INFINITY;
            for (int t = 16 * lane; t < min(n3, 16 * lane + 16); ++t) mx = fmaxf(mx, sm.m3[t]);
            sm.m4[lane] = mx;
        }
        // LSE: segment i's maximum is the maximum of its groups (the same float product
        // the segment used), merged with the segments' sums in float32.
        constexpr int per = (BF16 ? kSegTokensBf16 : kSegTokensF32) / 2048;  // level-3 blocks per segment
        float mi = -INFINITY, si = 0.f;
        if (lane < a.L.nseg) {
            float gmx = -INFINITY;
            for (int t = lane * per; t < min(n3, lane * per + per); ++t) gmx = fmaxf(gmx, sm.m3[t]);
            mi = gmx * c2;
            si = sm.part[lane];
        }
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) {
            const float om = __shfl_xor(mi, off);
            const float os = __shfl_xor(si, off);
            lse_combine(mi, si, om, os);
        }
        // row maximum over the level-3 maxima
        float rm = -INFINITY;
        for (int t = lane; t < n3; t += 64) rm = fmaxf(rm, sm.m3[t]);
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) rm = fmaxf(rm, __shfl_xor(rm, off));
        if (lane == 0) {
            const float lse = mi == -INFINITY ? -INFINITY : (mi + __builtin_amdgcn_logf(si)) * 0.69314718055994531f;
            if (r.kind == 0) {
                if (a.draft_lse) a.draft_lse[((size_t)r.b * a.K + r.k) * a.gamma + r.s] = lse;
            } else if (a.target_lse) {
                const size_t o = a.target_rows == 1 ? (size_t)r.b * (a.gamma + 1) + r.s
                                                    : ((size_t)r.b * a.K + r.k) * (a.gamma + 1) + r.s;
                a.target_lse[o] = lse;
            }
            sm.rowmax = rm;
            sm.n_l4 = sm.n_l3 = sm.n_l2 = sm.n_cand = 0;
            sm.n_ev[0] = sm.n_ev[1] = 0;
            sm.best_key = ordered_key(INFINITY);
            sm.key_min = 0x7FFFFFFF;
            sm.key_max = -1;
        }
    } else {
        // Context keys: the window's path tokens (published by earlier races of this
        // call, or inputs), both chains folded at once -- lane 0 this row's key, lane 1
        // the next depth's key up to its newest token (the winner of this race) --
        // then lane 0 waits for the key published by the race one depth up this path,
        // if any.
        const int tk = widx >= a.m ? path_token(a, r, widx - a.m, ep) : wtok;
        const uint64_t t = (uint64_t)(wpos + r.s) + (uint64_t)(lane == 1);
        uint32_t c0 = (uint32_t)a.key, c1 = (uint32_t)(a.key >> 32);
        const bool chain = (lane == 0 && prod < 0) || (lane == 1 && cons);
        if (chain) fold(c0, c1, (uint32_t)t, (uint32_t)(t >> 32), 0u);
        for (int i = 0; i < a.m; ++i) {
            const int w = __shfl(tk, lane == 0 ? i : a.m + i);
            if (chain && (lane == 0 || i + 1 < a.m)) fold(c0, c1, (uint32_t)w, (uint32_t)i, 1u);
        }
        if (lane == 0 && prod < 0) {
            sm.kappa0 = c0;
            sm.kappa1 = c1;
        }
        if (lane == 1 && cons) {
            sm.next0 = c0;
            sm.next1 = c1;
        }
        if (lane == 0 && prod >= 0) {
            const uint64_t* ks = (const uint64_t*)(a.ws + a.L.keys) + 2 * (size_t)prod;
            uint64_t w0 = ld_dev(ks), w1 = ld_dev(ks + 1);
            if ((uint32_t)(w0 >> 32) != ep) w0 = wait_slot(a, ks, ep);
            if ((uint32_t)(w1 >> 32) != ep) w1 = wait_slot(a, ks + 1, ep);
            sm.kappa0 = (uint32_t)w0;
            sm.kappa1 = (uint32_t)w1;
        }
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
        Row rs = r;
        rs.shift = sm.rowmax;
        race<BF16, VEC, LAYOUT>(a, rs, sm, gm, k0, k1);
    }
    if (tid == 0) {
        const int y = sm.win_token;
        if (cons) {
            uint32_t n0 = sm.next0, n1 = sm.next1;
            fold(n0, n1, (uint32_t)y, (uint32_t)(a.m - 1), 1u);
            uint64_t* ks = (uint64_t*)(a.ws + a.L.keys) + 2 * (size_t)r.row_id;
            st_dev(ks, ((uint64_t)ep << 32) | n0);
            st_dev(ks + 1, ((uint64_t)ep << 32) | n1);
        }
        st_dev((uint64_t*)(a.ws + a.L.tok) + r.row_id, ((uint64_t)ep << 32) | (uint32_t)y);
        if (r.kind == 0) {
            a.draft_tokens[((size_t)r.b * a.K + r.k) * a.gamma + r.s] = y;
        } else if (a.target_tokens) {
            const size_t o = a.target_rows == 1 ? (size_t)r.b * (a.gamma + 1) + r.s
                                                : ((size_t)r.b * a.K + r.k) * (a.gamma + 1) + r.s;
            a.target_tokens[o] = y;
        }
    }
    // The last row of a sequence in the work order walks its block.
    if (r.kind == a.walk_kind && r.s == a.walk_s && r.k == a.walk_k) walk(a, sm, r.b, ep);
    __builtin_amdgcn_s_setprio(0);
}

// ---------------------------------------------------------------- kernel

// Row and segment of a work item (phases of rows, each at one depth: its draft
// rows, then its target rows, each row segment by segment).
template <bool BF16>
__device__ __forceinline__ void decode_item(const RaceArgs& a, const Shared& sm, int item, Row& r, int& seg) {
    const size_t esize = BF16 ? 2 : 4;
    const int D = a.B * a.K * a.gamma;
    // the phase holding the item: the number of later phase starts at or below it
    // (phases start in increasing order; phase 0 starts at 0)
    static_assert(kMaxPhases <= 2 * 64, "phase starts fit two lanes per wave");
    const int lane = threadIdx.x & 63;
    const bool s0 = lane + 1 < a.n_phase && sm.ph_first[lane + 1] <= item;
    const bool s1 = lane + 65 < a.n_phase && sm.ph_first[lane + 65] <= item;
    const int ph = (int)__builtin_popcountll(__ballot(s0)) + (int)__builtin_popcountll(__ballot(s1));
    // (the item is uniform: the table entries are made scalar, so the divisions
    // below run on the scalar unit rather than on every lane)
    const int local = __builtin_amdgcn_readfirstlane(item) - __builtin_amdgcn_readfirstlane(sm.ph_first[ph]);
    const int rl = local / a.L.nseg;
    seg = local % a.L.nseg;
    const int d = __builtin_amdgcn_readfirstlane(sm.ph_depth[ph]);
    const int nd = __builtin_amdgcn_readfirstlane(sm.ph_nd[ph]);
    r.s = d;
    r.shift = 0.f;
    if (rl < nd) {
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
        const int rt = rl - nd;
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
        r.nslots = a.target_slots;
        r.invT = a.inv_T_target;
        r.T = a.T_target;
    }
}

// Four workgroups per CU (128 VGPRs).  Of every kRolePeriod blocks, kRoleFinish
// finish rows and the others only stream segments, so the streaming loop
// (software-pipelined) and the races neither share a loop nor wait for each other
// (the share of finishing blocks was measured: about 0.36 balances the two).  Both
// kinds take work in order from per-XCD queues (row R goes to queue R mod nq for
// both): streaming never waits, and a finishing workgroup waits only for segments
// (streamed without waiting) and for races of rows earlier in the order (taken
// earlier by running finishing workgroups), so every wait ends.
template <bool BF16, bool VEC, int LAYOUT>
__global__ __launch_bounds__(kBlock, 4) void race_kernel(RaceArgs a) {
    extern __shared__ __align__(16) unsigned char smem_raw[];
    Shared& sm = *reinterpret_cast<Shared*>(smem_raw);
    float* gm = reinterpret_cast<float*>(smem_raw + ((sizeof(Shared) + 15) & ~(size_t)15));
    const int tid = threadIdx.x;
    uint32_t* ctrl = ctrl_of(a);
    // roles: of every kRolePeriod consecutive blocks the last kRoleFinish finish rows
    // (the launch has at least kRolePeriod blocks); kRolePeriod is odd, so with
    // 8 kRolePeriod or more blocks every XCD queue (block mod 8) has both kinds
    const bool finisher = blockIdx.x % (unsigned)kRolePeriod >= (unsigned)(kRolePeriod - kRoleFinish);
    const int nq = gridDim.x >= 8u * kRolePeriod ? kMaxQueues : 1;
    const int q = (int)(blockIdx.x % (unsigned)nq);
    if (tid == 0) {
        sm.err_local = 0u;
        const uint32_t last = ld_dev(ctrl + kCtrlEpoch);
        sm.epoch = last == 0xFFFFFFFFu ? 1u : last + 1u;  // 1 .. 2^32-1
        sm.tick[0] = finisher ? take_row(a, q, nq) : take_item(a, q, nq);
    }
    for (int i = tid; i < a.n_phase; i += kBlock) {
        sm.ph_first[i] = a.phase_first[i];
        sm.ph_depth[i] = a.phase_depth[i];
        sm.ph_nd[i] = a.phase_nd[i];
    }
    __syncthreads();
    if (finisher) {
        // Before its first row, a finishing workgroup streams segments from its queue
        // until that row's segments are all taken: at the start the streaming is
        // behind and the first rows' races wait for it.  (It never waits here.)
        if (sm.tick[0] < a.n_rows) {
            const int last = sm.tick[0] * a.L.nseg + a.L.nseg - 1;
            for (int p = 0;; p ^= 1) {
                if (tid == 0) sm.tick[2 + p] = take_item(a, q, nq);
                __syncthreads();
                const int item = sm.tick[2 + p];
                if (item >= a.n_items) break;
                Row rs;
                int ss;
                decode_item<BF16>(a, sm, item, rs, ss);
                Unit<BF16, VEC> u[units_per_segment<BF16>()];
                issue_segment<BF16, VEC>(a, rs, ss, u);
                consume_segment<BF16, VEC>(a, rs, ss, sm, p, u);
                __syncthreads();
                publish_segment<BF16>(a, rs.row_id, ss, sm, p);
                if (item >= last) break;
            }
        }
        for (int R = sm.tick[0]; R < a.n_rows;) {
            Row r;
            int seg;
            decode_item<BF16>(a, sm, R * a.L.nseg + a.L.nseg - 1, r, seg);
            finish_row<BF16, VEC, LAYOUT>(a, r, sm, gm);
            if (tid == 0) sm.tick[0] = take_row(a, q, nq);
            __syncthreads();
            R = sm.tick[0];
        }
    } else {
        // Software-pipelined: the next segment's loads are issued before the current
        // one is published.
        Unit<BF16, VEC> u[units_per_segment<BF16>()];
        int item = sm.tick[0], seg = 0;
        Row r;
        if (item < a.n_items) {
            decode_item<BF16>(a, sm, item, r, seg);
            issue_segment<BF16, VEC>(a, r, seg, u);
        }
        for (int parity = 0; item < a.n_items; parity ^= 1) {
            if (tid == 0) sm.tick[parity ^ 1] = take_item(a, q, nq);
            consume_segment<BF16, VEC>(a, r, seg, sm, parity, u);
            __syncthreads();
            const int pub_row = r.row_id, pub_seg = seg;
            item = sm.tick[parity ^ 1];
            if (item < a.n_items) {
                decode_item<BF16>(a, sm, item, r, seg);
                issue_segment<BF16, VEC>(a, r, seg, u);
            }
            publish_segment<BF16>(a, pub_row, pub_seg, sm, parity);
        }
    }
    // The last workgroup to leave resets the queues, hands over the call's error bits
    // and advances the epoch.  A workgroup that recorded errors fences (release)
    // before it counts its exit, and the last one fences (acquire) after it: its
    // read of the call's bits then sees every error of the call.  The exit count
    // itself stays relaxed (a release per workgroup writes back its L2: ~19 us).
    __syncthreads();
    if (tid == 0) {
        if (sm.err_local) __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
        const uint32_t old = __hip_atomic_fetch_add(ctrl + kCtrlExited, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (old == gridDim.x - 1) {
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
            const uint32_t bits =
                __hip_atomic_exchange(ctrl + kCtrlCallErrors, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (bits) __hip_atomic_fetch_or(ctrl + kCtrlErrors, bits, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (a.status) *a.status = bits;
            for (int i = 0; i < 2 * kMaxQueues; ++i) st_dev(ctrl + ctrl_queue(i), 0u);
            st_dev(ctrl + kCtrlExited, 0u);
            st_dev(ctrl + kCtrlEpoch, sm.epoch);
        }
    }
}

// Shared, the group maxima and the level-4 list (K slots x level-4 nodes, 256 groups
// each), in the order level4_list assumes.
size_t shared_bytes(int ng, int K) {
    return ((sizeof(Shared) + 15) & ~(size_t)15) + (size_t)((ng + 3) & ~3) * sizeof(float) +
           (size_t)K * (size_t)((ng + 255) / 256) * sizeof(Node);
}

template <bool BF16, bool VEC, int LAYOUT>
hipError_t launch_one(const RaceArgs& a, hipStream_t stream) {
    const size_t smem = shared_bytes(a.L.ng, a.K);
    auto fn = race_kernel<BF16, VEC, LAYOUT>;
    int per_cu = 0;
    hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kBlock, smem);
    if (e != hipSuccess) return e;
    int dev = 0, cus = 0;
    if ((e = hipGetDevice(&dev)) != hipSuccess) return e;
    if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess) return e;
    if (per_cu < 1) per_cu = 1;
    // both kinds of workgroup: at least kRolePeriod blocks
    long grid = (long)per_cu * cus;
    if (grid > (long)kRolePeriod * a.n_items) grid = (long)kRolePeriod * a.n_items;
    if (grid < kRolePeriod) grid = kRolePeriod;
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


// ---------------------------------------------------------------- static scratch

// The allocation-free entry point's workspace: one fixed array per device, held
// until the process ends.  In host code `scratch` is only a handle for the
// runtime; its device address is looked up once per device (with that device
// current) and kept, and only that address is passed to kernels.
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

hipError_t static_scratch(void** out, hipStream_t stream) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        if ((e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch))) != hipSuccess) return e;
        if (!p || ((uintptr_t)p & 255u) != 0) return hipErrorInvalidSymbol;
        // zero once (control words, epoch, queues) with a fill kernel ahead of the
        // first call on the caller's stream
        if ((e = launch_fill_zero((uint32_t*)p, kStaticScratchBytes / 4, stream)) != hipSuccess) return e;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return hipSuccess;
}

}  // namespace psd
