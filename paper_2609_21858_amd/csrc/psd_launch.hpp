// psd_launch.hpp -- host-side launchers of the HIP kernels (internal to libpsd).
#pragma once

#include <hip/hip_runtime.h>

#include "psd_layout.hpp"

namespace psd {

// Control word that carries the race kernel's share of a call's error bits to a
// later walk kernel of the same call (a word the race kernel uses for nothing else).
constexpr int kCtrlRaceBits = 7;
// Epoch of the last identical-drafter launch that ran every depth, and its workgroups
// that have left (words of their own: the race kernel may run beside it).
constexpr int kCtrlMpfrEpoch = 8;
constexpr int kCtrlMpfrExited = 9;

struct DetectArgs {
    const int32_t* tokens;  // [n_seq][row_stride], positions [0, seq_len) of each row scored
    const int32_t* n0;      // [n_seq]
    double* out_score;      // [n_seq] (Aaronson's S_A only) or [n_seq][4] (every score)
    int32_t* out_count;     // [n_seq]
    float* out_per_token;   // nullable [n_seq][seq_len]
    uint64_t key;
    int n_seq, seq_len, V, K, m;
    int row_stride;
    // further scores (App. on Li et al.'s and Lattimore's scores), with multi = 1
    int multi;
    double li_lnk, li_a, li_b;  // ln k_Delta, Delta / (1 - Delta), (1 - q) / q
    int li_q;                   // q_Delta > 0
    double pl_cap, pl_c0;       // eps^{-1/2}, 2 - sqrt(eps)
};

// Null-tail p-values of the four detection scores of each sequence.
struct ScorePvalueArgs {
    const double* scores;   // [n][4]: S_A, S_U, S_Li, S_PL
    const int32_t* count;   // [n]
    double* out_log_p;      // [n][4]
    int n;
    double li_lnk, li_a, li_b;
    int li_q;
    double pl_cap, pl_c0, pl_eps;
};
hipError_t launch_score_pvalues(const ScorePvalueArgs& a, hipStream_t stream);
hipError_t launch_detection_rate(int n, const double* log_p, int stride, double log_alpha, int32_t* out_count,
                                 hipStream_t stream);

// One depth of drafting with identical drafters (multi-sample PFR), one workgroup
// per draft row (b, k) of depth s.
struct MpfrArgs {
    const void* logits;         // [B][K][s_count][V] draft rows of depths s_begin .. s_begin + s_count - 1
    int32_t* draft_tokens;      // [B][K][gamma]: depths < s read, depth s written
    float* draft_lse;           // nullable [B][K][gamma]
    const int32_t* prefix;      // [B][m]
    const int64_t* start_pos;   // [B]
    uint32_t* ctrl;             // workspace control words (error bits of the call)
    uint64_t key;
    int V, K, m, B, gamma;
    int s_begin, s_count, s;    // depth of this launch: s_begin <= s < s_begin + s_count
    float T, invT;
    // Written by the streaming launch and read by the sampling launches, each word
    // (epoch << 32) | payload (draft row ids): a sampling launch that runs every depth
    // may run beside the streaming launch and waits for the tags.
    uint64_t* row_gm;           // [B*K*gamma][groups] group maxima of the draft rows (float bits)
    uint64_t* row_max;          // [B*K*gamma] their maxima (float bits)
    uint64_t* row_seed;         // [B*K*gamma][8] their seed tokens (-1: none)
    uint64_t* tok_slot;         // nullable [B*K*gamma]: the drafts of a launch that runs every
                                // depth, as (epoch << 32) | token, for the later depths' waits
    uint32_t spin_limit;        // polls of a bounded wait before it gives up
    int stream_records_epoch;   // the streaming launch records its epoch (no sampling launch
                                // that runs every depth follows it to do so)
    int stream_grid;            // workgroups of the streaming launch (0: one per row); each
                                // streams rows blockIdx.x, blockIdx.x + grid, ... (depth-major)
};

// Identical drafters: the draft rows' group maxima and maxima, streamed once per call
// ahead of the depth-by-depth sampling, after the race kernel's workspace, then the
// shared target chain's tokens for a walk kernel that runs after the drafts.
struct MpfrLayout {
    size_t gm, rmax, seed, slot, ytok, total;
};
// Identical-drafter calls with fewer than this many (sequence, path) workgroups per
// depth stream their draft rows in a launch of their own; larger ones stream each
// depth's rows in its sampling launch.
constexpr long kMpfrStreamBelow = 1024;

inline MpfrLayout mpfr_layout(const WsLayout& L, int B, int K, int gamma) {
    MpfrLayout M;
    // the streamed rows' words exist only when the call has a streaming launch
    const size_t rows = (long)B * K < kMpfrStreamBelow ? (size_t)B * K * gamma : 0;
    M.gm = L.total;
    M.rmax = align256(M.gm + rows * (size_t)L.ng * 8);
    M.seed = align256(M.rmax + rows * 8);
    M.slot = align256(M.seed + rows * 8 * 8);  // 8 seeds per row
    M.ytok = align256(M.slot + rows * 8);      // one tagged draft per row
    M.total = align256(M.ytok + (size_t)B * (gamma + 1) * 4);  // shared-chain targets [B][gamma+1]
    return M;
}

// Truncation before the race (top-k, then top-p): per row a kept list of at most
// top_k (token, logit) pairs, sorted, its length and LSE, after the race kernel's
// workspace (same row identifiers).
constexpr int kMaxTopK = 256;
struct TopkLayout {
    size_t tok, val, len, lse, chain, total;  // offsets from the workspace base; total = end
};
inline TopkLayout topk_layout(const WsLayout& L, int top_k) {
    TopkLayout T;
    size_t o = L.total;
    T.tok = o;
    o = align256(o + (size_t)L.n_rows * top_k * 4);
    T.val = o;
    o = align256(o + (size_t)L.n_rows * top_k * 4);
    T.len = o;
    o = align256(o + (size_t)L.n_rows * 4);
    T.lse = o;
    o = align256(o + (size_t)L.n_rows * 4);
    T.chain = o;  // shared target chain tokens [B][gamma + 1] (n_rows >= B (gamma + 1))
    o = align256(o + (size_t)L.n_rows * 4);
    T.total = o;
    return T;
}

// One launch selects the kept lists of up to two row segments (the draft rows and the
// target rows of a call): blocks [0, seg[0].n_rows) take segment 0, the next
// seg[1].n_rows blocks segment 1.  Row r of a segment is row id
// row_id_base + (group > 0 ? (r / group) * group_stride + r % group : r), and its LSE
// goes to lse_out[lse_index_base + (same map with lse_group_stride)] when non-null.
struct TopkSegment {
    const void* logits;  // [n_rows][V]
    int n_rows;
    float T;
    int row_id_base, group, group_stride;
    float* lse_out;
    int lse_index_base, lse_group_stride;
};
struct TopkSelectArgs {
    TopkSegment seg[2];
    int V;
    int top_k;
    float top_p;
    int cap;
    int32_t* list_tok;
    float* list_val;
    int32_t* list_len;
    float* list_lse;
    uint32_t* radix_rows;  // nullable: counts rows whose one-pass selection could not be
                           // proven exact and were selected again by radix passes
};

struct TopkRaceArgs {
    const int32_t* prefix;
    const int64_t* start_pos;
    int32_t* draft_tokens;   // [B][K][gamma]
    int32_t* out_tokens;     // [B][gamma+1] (target_rows > 0)
    int32_t* out_len;        // [B]
    int32_t* target_tokens;  // nullable
    const int32_t* list_tok;
    const float* list_val;
    const int32_t* list_len;
    int cap;
    uint64_t key;
    int V, K, m, B, gamma;
    int s_begin, s_count;    // draft depths of this call
    int target_rows;         // 0 (drafting only), 1, K
    int mpfr;
    float T_target, T_draft;
    int target_waves;        // waves sharing each shared-chain target race (set by the launcher)
    int32_t* chain;          // workspace [B][gamma + 1]: shared-chain targets for the walk kernel
    uint32_t* ctrl;          // workspace control words (the call's error bits)
    uint32_t* status;        // nullable: the call's error bits for the caller
    const uint32_t* status_in;  // nullable: bits already taken from the call by an earlier
                                // kernel of the same call, added to *status
};

// Position-indexed toy language model: target rows [B][gamma+1][V] at positions
// start_pos[b] + s and draft rows [B][K][gamma][V] (nullable).
struct ToyArgs {
    const int64_t* start_pos;
    void* target_logits;
    void* draft_logits;
    uint64_t seed, draft_seed;
    float sigma, w;      // noise scale; weight of the rank term (-alpha ln 2 / 2^23)
    float tau0, tau1;    // draft noise of sequences b < tau_split, and of the others
    int tau_split;
    int V, K, B, gamma;
};

// Commit one block's emitted tokens into the texts (out_len NULL: first block, from
// the prompts), then the next block's start positions, windows and active count.
struct AdvanceArgs {
    const int32_t* out_tokens;  // [B][gamma+1]
    const int32_t* out_len;     // [B], nullable
    int32_t* text;              // [B][text_stride]
    int64_t text_stride;
    int64_t* length;            // [B]
    int64_t* start_pos;         // [B]
    int32_t* prefix;            // [B][m]
    int32_t* n_active;          // one word
    int B, gamma, m;
    int64_t max_len;
};

hipError_t launch_toy_rows(const ToyArgs& a, bool bf16, hipStream_t stream);
hipError_t launch_advance(const AdvanceArgs& a, hipStream_t stream);
hipError_t launch_topk_select(const TopkSelectArgs& a, bool bf16, hipStream_t stream);
hipError_t launch_topk_race(const TopkRaceArgs& a, int layout, hipStream_t stream);
// The walk alone (one thread per sequence) over shared-chain targets a.chain
// [B][gamma+1] and the drafts, then the call's error bits (with *a.status_in).
hipError_t launch_walk(const TopkRaceArgs& a, hipStream_t stream);

hipError_t launch_race(const RaceArgs& a, bool bf16, bool vec, int layout, hipStream_t stream);
// The sampling of depths [s_begin, s_begin + s_count): one launch that runs every
// depth when the drafts can be handed over in tagged slots (tok_slot set, more than
// one depth) and every workgroup of it can be resident at once, else one launch per
// depth.
hipError_t launch_mpfr_depths(MpfrArgs a, bool bf16, bool vec, int layout, hipStream_t stream);
// Whether one sampling launch can run every depth of a: more than one depth, and all
// B K workgroups resident together.  *fits is set; a HIP error of the query is returned.
hipError_t mpfr_all_depths_fit(const MpfrArgs& a, bool bf16, bool vec, int layout, bool* fits);
hipError_t launch_mpfr_stream(const MpfrArgs& a, bool bf16, bool vec, hipStream_t stream);
hipError_t launch_finish_status(uint32_t* ctrl, uint32_t* status, hipStream_t stream);
hipError_t launch_detect(const DetectArgs& a, int layout, hipStream_t stream);
hipError_t launch_pvalue(int n, const double* score, const int32_t* count, double* out_log_p,
                         double* out_anlppt, hipStream_t stream);
hipError_t launch_philox(int n, const uint32_t* ctr, const uint32_t* key, uint32_t* out, hipStream_t stream);
hipError_t launch_context_keys(uint64_t key, int m, int n, const int64_t* t, const int32_t* windows,
                               uint32_t* out, hipStream_t stream);
hipError_t launch_clock_values(int layout, int V, int n, const uint32_t* kappa, const int32_t* slot,
                               const int32_t* token, double* out, hipStream_t stream);
hipError_t launch_fill_zero(uint32_t* p, size_t n_words, hipStream_t stream);

// Bytes of the fixed per-device scratch behind psd_verify_static.
constexpr size_t kStaticScratchBytes = size_t(32) << 20;
// Device address of this device's fixed scratch (looked up and zeroed on the first
// call on the device, the clear enqueued on `stream`).
hipError_t static_scratch(void** out, hipStream_t stream);

}  // namespace psd
