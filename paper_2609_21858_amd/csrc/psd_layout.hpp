// psd_layout.hpp -- workspace layout and kernel arguments of the fused race kernel
// (host and device).
#pragma once

#include <stddef.h>
#include <stdint.h>

namespace psd {

constexpr int kBlock = 256;             // threads per workgroup (4 wave64)
constexpr int kSegTokensBf16 = 16384;   // tokens per work item: 32 KiB of bf16
constexpr int kSegTokensF32 = 8192;     // 32 KiB of float32
constexpr int kMaxDepth = 33;           // gamma + 1 <= 33
constexpr int kMaxPhases = 2 * kMaxDepth;

inline int seg_tokens(int dtype_bf16) { return dtype_bf16 ? kSegTokensBf16 : kSegTokensF32; }

// Control words at the start of every workspace (fixed positions for every call shape).
constexpr int kCtrlWords = 2048;   // 8 KiB
constexpr int kCtrlExited = 1;     // workgroups that left the kernel
constexpr int kCtrlErrors = 2;     // sticky error bits (since the last clear)
constexpr int kCtrlCallErrors = 3; // error bits of the running call; moved to kCtrlErrors and the
                                   // caller's status word by the call's last workgroup
constexpr int kCtrlEpoch = 5;      // epoch of the last completed call
constexpr int kCtrlTopkRadix = 6;  // rows of truncated calls selected by radix passes (cumulative)
constexpr int kMaxQueues = 8;      // work queues (one per XCD) of each kind, counters 256 B apart
// counter of segment queue q (q < kMaxQueues) or of row queue q - kMaxQueues
inline constexpr int ctrl_queue(int q) { return 64 * (q + 1); }

// Every slot a call publishes is (epoch << 32) | 32-bit payload, with the call's
// epoch (1 .. 2^32-1) in the same bits for every slot kind, so readers detect fresh
// data by its tag, stale data of another call shape never matches, and nothing is
// cleared between calls:
//   tok  : payload = int32 token
//   part : payload = float bits of the segment's sum of exp2 (relative to its max)
//   gmax : payload = float bits of the group's maximum logit
//   m3   : payload = float bits of a 2048-token block's maximum logit
//   stop : payload = int32 index of the segment's largest group (lowest index; -1: none)
//   keys : two slots per row, payload = the two words of the context key of the
//          next depth of the row's path (published by the row's race)
//
// Row identifiers (independent of the call):
//   draft (b, k, s)            : (b*K + k)*gamma + s
//   target shared (b, s)       : D + b*(gamma+1) + s                 D = B*K*gamma
//   target per path (b, k, s)  : D + (b*K + k)*(gamma+1) + s
struct WsLayout {
    size_t ctrl;  // uint32[kCtrlWords]
    size_t tok;   // uint64[n_rows]
    size_t part;  // uint64[n_rows][nseg]
    size_t gmax;  // uint64[n_rows][ng]
    size_t m3;    // uint64[n_rows][n3]
    size_t stop;  // uint64[n_rows][nseg]
    size_t keys;  // uint64[n_rows][2]
    size_t total;
    int n_rows, nseg, ng, n3;
};

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

inline WsLayout ws_layout(int B, int K, int gamma, int V, int dtype_bf16) {
    WsLayout L;
    const long D = (long)B * K * gamma;
    L.n_rows = (int)(D + (long)B * K * (gamma + 1));
    L.nseg = (V + seg_tokens(dtype_bf16) - 1) / seg_tokens(dtype_bf16);
    L.ng = (V + 127) / 128;
    L.n3 = (V + 2047) / 2048;
    size_t o = 0;
    L.ctrl = o;
    o = align256(o + kCtrlWords * 4);
    L.tok = o;
    o = align256(o + (size_t)L.n_rows * 8);
    L.part = o;
    o = align256(o + (size_t)L.n_rows * L.nseg * 8);
    L.gmax = o;
    o = align256(o + (size_t)L.n_rows * L.ng * 8);
    L.m3 = o;
    o = align256(o + (size_t)L.n_rows * L.n3 * 8);
    L.stop = o;
    o = align256(o + (size_t)L.n_rows * L.nseg * 8);
    L.keys = o;
    o = align256(o + (size_t)L.n_rows * 16);
    L.total = o;
    return L;
}

struct RaceArgs {
    const void* draft_logits;   // [B][K][s_count][V] or null
    const void* target_logits;  // [B][gamma+1][V] or [B][K][gamma+1][V] or null
    const int32_t* prefix;      // [B][m]
    const int64_t* start_pos;   // [B]
    int32_t* draft_tokens;      // [B][K][gamma]
    int32_t* out_tokens;        // [B][gamma+1] or null
    int32_t* out_len;           // [B] or null
    float* target_lse;          // nullable
    float* draft_lse;           // nullable
    int32_t* target_tokens;     // nullable
    unsigned char* ws;          // workspace base
    WsLayout L;
    uint64_t key;
    int V, K, m, B, gamma;
    float T_target, T_draft;    // temperatures
    float inv_T_target, inv_T_draft;
    int s_begin, s_count;       // draft depths computed in this call (s_count = 0: none)
    int target_rows;            // 0: no target rows, 1: shared, K: per path
    int target_slots;           // slots a target row races: K (distinct drafters), 1 (identical: MPFR)
    int n_items;                // rows * nseg
    int n_rows;                 // rows of this call
    // Work order: phases of rows, each at one depth: phase_nd draft rows, then
    // phase_nt target rows; a phase's items start at phase_first.
    int n_phase;
    int phase_first[kMaxPhases];
    int phase_depth[kMaxPhases];
    int phase_nd[kMaxPhases];
    int phase_nt[kMaxPhases];
    // the row of each sequence that walks its block: (kind, depth, path); kind -1: none
    int walk_kind, walk_s, walk_k;
    uint32_t* status;     // nullable: this call's error bits, written by its last workgroup
    uint32_t spin_limit;  // polls of a bounded wait before it gives up (psd_set_spin_limit)
};

}  // namespace psd
