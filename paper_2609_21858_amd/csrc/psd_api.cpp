// psd_api.cpp -- C ABI of libpsd: argument validation, workspace sizing and launches.
// Every argument is checked before anything is enqueued; no exception crosses the ABI.
#include <hip/hip_runtime.h>

#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <mutex>

#include "../../include/psd.h"
#include "psd_launch.hpp"
#include "psd_layout.hpp"

namespace {

thread_local char g_err[512] = "";

// Polls of a bounded cross-workgroup wait before it gives up (test hook, psd_set_spin_limit).
constexpr uint32_t kDefaultSpinLimit = 1u << 22;
std::atomic<uint32_t> g_spin_limit{kDefaultSpinLimit};

// A side stream and a fork and a join event per device, created on first use and
// kept until the process ends.  They let an identical-drafter call race its
// target chain beside its drafting launches.  The mutex is held from the fork's
// record to the join's wait, so calls from several host threads never mix up
// their events.
constexpr int kMaxForkDevices = 64;
struct Fork {
    hipStream_t side;
    hipEvent_t in, out;
};
std::mutex g_fork_mu;
Fork g_fork[kMaxForkDevices] = {};

// The current device's fork objects (the caller holds g_fork_mu), or nullptr if they
// cannot be created.
Fork* fork_objects() {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxForkDevices) return nullptr;
    Fork& f = g_fork[dev];
    if (!f.side) {
        hipStream_t st = nullptr;
        hipEvent_t e0 = nullptr, e1 = nullptr;
        if (hipStreamCreateWithFlags(&st, hipStreamNonBlocking) != hipSuccess) return nullptr;
        if (hipEventCreateWithFlags(&e0, hipEventDisableTiming) != hipSuccess ||
            hipEventCreateWithFlags(&e1, hipEventDisableTiming) != hipSuccess) {
            if (e0) (void)hipEventDestroy(e0);
            (void)hipStreamDestroy(st);
            return nullptr;
        }
        f.in = e0;
        f.out = e1;
        f.side = st;
    }
    return &f;
}

psd_status fail(psd_status st, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return st;
}

psd_status hip_fail(hipError_t e, const char* where) {
    return fail(PSD_E_HIP, "%s: %s", where, hipGetErrorString(e));
}

psd_status check_params(const psd_params* p) {
    if (!p) return fail(PSD_E_ARG, "params is NULL");
    if (p->vocab < 1 || p->vocab > PSD_MAX_VOCAB) return fail(PSD_E_ARG, "vocab %d outside [1, %d]", p->vocab, PSD_MAX_VOCAB);
    if (p->num_drafts < 1 || p->num_drafts > PSD_MAX_DRAFTS)
        return fail(PSD_E_ARG, "num_drafts %d outside [1, %d]", p->num_drafts, PSD_MAX_DRAFTS);
    if (p->ctx_window < 0 || p->ctx_window > PSD_MAX_WINDOW)
        return fail(PSD_E_ARG, "ctx_window %d outside [0, %d]", p->ctx_window, PSD_MAX_WINDOW);
    if (!(p->temp_target > 0.f) || !isfinite(p->temp_target))
        return fail(PSD_E_ARG, "temp_target must be finite and > 0");
    if (!(p->temp_draft > 0.f) || !isfinite(p->temp_draft)) return fail(PSD_E_ARG, "temp_draft must be finite and > 0");
    if (p->dtype != PSD_F32 && p->dtype != PSD_BF16) return fail(PSD_E_ARG, "unknown dtype %d", p->dtype);
    if (p->clocks != PSD_CLOCKS_TREE && p->clocks != PSD_CLOCKS_FLAT)
        return fail(PSD_E_ARG, "unknown clock layout %d", p->clocks);
    if (p->mode != PSD_MODE_HET && p->mode != PSD_MODE_MPFR) return fail(PSD_E_ARG, "unknown mode %d", p->mode);
    if (p->top_k < 0 || p->top_k > PSD_MAX_TOP_K) return fail(PSD_E_ARG, "top_k %d outside [0, %d]", p->top_k, PSD_MAX_TOP_K);
    if (!(p->top_p > 0.f && p->top_p <= 1.f)) return fail(PSD_E_ARG, "top_p must be in (0, 1]");
    if (p->top_p < 1.f && p->top_k == 0) return fail(PSD_E_ARG, "top_p < 1 needs top_k in [1, %d]", PSD_MAX_TOP_K);
    return PSD_OK;
}

// Bytes a block of these parameters needs: the race kernel's workspace, plus the kept
// lists of every row when logits are truncated.
size_t workspace_need(const psd_params* p, int B, int gamma) {
    const psd::WsLayout L = psd::ws_layout(B, p->num_drafts, gamma, p->vocab, p->dtype == PSD_BF16);
    if (p->top_k > 0) return psd::topk_layout(L, p->top_k).total;
    if (p->mode == PSD_MODE_MPFR) return psd::mpfr_layout(L, B, p->num_drafts, gamma).total;
    return L.total;
}

psd_status check_block(const psd_params* p, const psd_block* b) {
    if (!b) return fail(PSD_E_ARG, "block is NULL");
    if (b->batch < 1 || b->batch > PSD_MAX_BATCH) return fail(PSD_E_ARG, "batch %d outside [1, %d]", b->batch, PSD_MAX_BATCH);
    if (b->gamma < 1 || b->gamma > PSD_MAX_GAMMA) return fail(PSD_E_ARG, "gamma %d outside [1, %d]", b->gamma, PSD_MAX_GAMMA);
    if (!b->start_pos) return fail(PSD_E_ARG, "start_pos is NULL");
    if (p->ctx_window > 0 && !b->prefix_tokens) return fail(PSD_E_ARG, "prefix_tokens is NULL with ctx_window > 0");
    const psd::WsLayout L = psd::ws_layout(b->batch, p->num_drafts, b->gamma, p->vocab, p->dtype == PSD_BF16);
    const long items = (long)L.n_rows * L.nseg;
    if (items > 0x7FFFFFFFL) return fail(PSD_E_ARG, "block too large (%ld work items)", items);
    if (!b->workspace) return fail(PSD_E_WORKSPACE, "workspace is NULL");
    const size_t need = workspace_need(p, b->batch, b->gamma);
    if (b->workspace_bytes < need)
        return fail(PSD_E_WORKSPACE, "workspace has %zu bytes, needs %zu", b->workspace_bytes, need);
    if (((uintptr_t)b->workspace & 255u) != 0) return fail(PSD_E_WORKSPACE, "workspace must be 256-byte aligned");
    return PSD_OK;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

psd::RaceArgs base_args(const psd_params* p, const psd_block* b) {
    psd::RaceArgs a;
    memset(&a, 0, sizeof a);
    a.prefix = b->prefix_tokens;
    a.start_pos = b->start_pos;
    a.ws = (unsigned char*)b->workspace;
    a.L = psd::ws_layout(b->batch, p->num_drafts, b->gamma, p->vocab, p->dtype == PSD_BF16);
    a.key = p->key;
    a.V = p->vocab;
    a.K = p->num_drafts;
    a.m = p->ctx_window;
    a.B = b->batch;
    a.gamma = b->gamma;
    a.T_target = p->temp_target;
    a.T_draft = p->temp_draft;
    a.inv_T_target = 1.0f / p->temp_target;
    a.inv_T_draft = 1.0f / p->temp_draft;
    a.status = b->status;
    a.spin_limit = g_spin_limit.load(std::memory_order_relaxed);
    a.target_slots = p->mode == PSD_MODE_MPFR ? 1 : p->num_drafts;
    return a;
}

// Work order.  Every row comes after the rows whose races it waits for.  With a
// shared target chain and drafts in the same call, the two chains are
// independent: the target chain, one depth longer, is queued one depth ahead of
// the drafts, so its waits overlap draft streaming, and each sequence's last
// draft row walks its block.  Otherwise rows go depth by depth, drafts before targets.
void build_depths(psd::RaceArgs& a, int n_depth) {
    int first = 0, n = 0;
    auto add = [&](int d, int nd, int nt) {
        if (nd + nt == 0) return;
        a.phase_first[n] = first;
        a.phase_depth[n] = d;
        a.phase_nd[n] = nd;
        a.phase_nt[n] = nt;
        first += (nd + nt) * a.L.nseg;
        ++n;
    };
    const bool targets_first = a.target_rows == 1 && a.s_count > 0;
    if (targets_first) {
        // the target chain runs one depth ahead: t0 t1 d0 t2 d1 ... t_gamma d_(gamma-1)
        int dt = 0;
        for (int d = a.s_begin; d < a.s_begin + a.s_count; ++d) {
            while (dt <= a.gamma && dt <= d + 1) add(dt++, 0, a.B);
            add(d, a.B * a.K, 0);
        }
        while (dt <= a.gamma) add(dt++, 0, a.B);
        a.walk_kind = 0;
        a.walk_s = a.s_begin + a.s_count - 1;
        a.walk_k = a.K - 1;
    } else {
        for (int d = 0; d < n_depth; ++d) {
            const int nd = (a.s_count > 0 && d >= a.s_begin && d < a.s_begin + a.s_count) ? a.B * a.K : 0;
            const int nt = (a.target_rows > 0 && d <= a.gamma) ? a.B * a.target_rows : 0;
            add(d, nd, nt);
        }
        a.walk_kind = a.target_rows > 0 ? 1 : -1;
        a.walk_s = a.gamma;
        a.walk_k = a.target_rows == 1 ? 0 : a.K - 1;
    }
    a.n_phase = n;
    a.n_items = first;
    a.n_rows = first / a.L.nseg;
}

// Identical drafters: depths [s_begin, s_begin + s_count) drafted one launch per depth
// (each depth's contexts depend on the previous depth's drafts).  mpfr_args fills
// the arguments, mpfr_stream_rows launches the call's streaming pass when there is
// one, mpfr_sample_depths the depth launches.
psd::MpfrArgs mpfr_args(const psd_params* p, const psd_block* b, int32_t s_begin, int32_t s_count,
                        const void* draft_logits, int32_t* draft_tokens, float* draft_lse) {
    psd::MpfrArgs m;
    memset(&m, 0, sizeof m);
    m.logits = draft_logits;
    m.draft_tokens = draft_tokens;
    m.draft_lse = draft_lse;
    m.prefix = b->prefix_tokens;
    m.start_pos = b->start_pos;
    m.ctrl = (uint32_t*)((unsigned char*)b->workspace +
                         psd::ws_layout(b->batch, p->num_drafts, b->gamma, p->vocab, p->dtype == PSD_BF16).ctrl);
    m.key = p->key;
    m.V = p->vocab;
    m.K = p->num_drafts;
    m.m = p->ctx_window;
    m.B = b->batch;
    m.gamma = b->gamma;
    m.s_begin = s_begin;
    m.s_count = s_count;
    m.T = p->temp_draft;
    m.invT = 1.0f / p->temp_draft;
    m.spin_limit = g_spin_limit.load(std::memory_order_relaxed);
    return m;
}

bool mpfr_vec(const psd_params* p, const void* draft_logits) {
    const size_t es = p->dtype == PSD_BF16 ? 2 : 4;
    return ((size_t)p->vocab * es) % 16 == 0 && aligned16(draft_logits);
}

// A depth's launch has one workgroup per (sequence, path), each streaming its row.
// When those cannot fill the device (B K < 1024), every draft row of the call is
// streamed first in one launch (group maxima, maxima, LSE) and the depths only sample
// (in one launch when its workgroups fit the device together); otherwise each depth's
// streaming overlaps its contexts' sampling.
// Sets the streamed rows' words and the form of the sampling (one launch for every
// depth when it fits the device, else one per depth); *streamed tells whether the call
// has a streaming launch.
psd_status mpfr_prepare(const psd_params* p, const psd_block* b, psd::MpfrArgs& m, bool* streamed) {
    *streamed = (long)b->batch * p->num_drafts < psd::kMpfrStreamBelow;
    if (!*streamed) return PSD_OK;
    const psd::WsLayout L = psd::ws_layout(b->batch, p->num_drafts, b->gamma, p->vocab, p->dtype == PSD_BF16);
    const psd::MpfrLayout M = psd::mpfr_layout(L, b->batch, p->num_drafts, b->gamma);
    m.row_gm = (uint64_t*)((unsigned char*)b->workspace + M.gm);
    m.row_max = (uint64_t*)((unsigned char*)b->workspace + M.rmax);
    m.row_seed = (uint64_t*)((unsigned char*)b->workspace + M.seed);
    bool fits = false;
    hipError_t e = psd::mpfr_all_depths_fit(m, p->dtype == PSD_BF16, mpfr_vec(p, m.logits), p->clocks, &fits);
    if (e != hipSuccess) return hip_fail(e, "MPFR occupancy query");
    m.tok_slot = fits ? (uint64_t*)((unsigned char*)b->workspace + M.slot) : nullptr;
    m.stream_records_epoch = fits ? 0 : 1;
    return PSD_OK;
}

psd_status mpfr_stream_rows(const psd_params* p, psd::MpfrArgs& m, hipStream_t stream) {
    hipError_t e = psd::launch_mpfr_stream(m, p->dtype == PSD_BF16, mpfr_vec(p, m.logits), stream);
    if (e != hipSuccess) return hip_fail(e, "MPFR stream kernel launch");
    return PSD_OK;
}

psd_status mpfr_sample_depths(const psd_params* p, psd::MpfrArgs& m, hipStream_t stream) {
    hipError_t e = psd::launch_mpfr_depths(m, p->dtype == PSD_BF16, mpfr_vec(p, m.logits), p->clocks, stream);
    if (e != hipSuccess) return hip_fail(e, "MPFR draft kernel launch");
    return PSD_OK;
}

psd_status run_mpfr_drafts(const psd_params* p, const psd_block* b, int32_t s_begin, int32_t s_count,
                           const void* draft_logits, int32_t* draft_tokens, float* draft_lse, hipStream_t stream) {
    psd::MpfrArgs m = mpfr_args(p, b, s_begin, s_count, draft_logits, draft_tokens, draft_lse);
    bool streamed = false;
    psd_status st = mpfr_prepare(p, b, m, &streamed);
    if (st == PSD_OK && streamed) st = mpfr_stream_rows(p, m, stream);
    if (st != PSD_OK) return st;
    return mpfr_sample_depths(p, m, stream);
}

// Truncated logits: the kept list of every row of the call, then one workgroup per
// sequence racing the lists (drafts of depths [s_begin, s_begin + s_count), then the
// target rows when target_rows > 0, then the walk).
psd_status run_topk(const psd_params* p, const psd_block* b, int32_t s_begin, int32_t s_count, int32_t target_rows,
                    const void* target_logits, const void* draft_logits, int32_t* draft_tokens, int32_t* out_tokens,
                    int32_t* out_len, float* target_lse, float* draft_lse, int32_t* target_tokens, hipStream_t stream) {
    const bool bf16 = p->dtype == PSD_BF16;
    const psd::WsLayout L = psd::ws_layout(b->batch, p->num_drafts, b->gamma, p->vocab, bf16);
    const psd::TopkLayout T = psd::topk_layout(L, p->top_k);
    unsigned char* ws = (unsigned char*)b->workspace;
    const int K = p->num_drafts, G = b->gamma, B = b->batch;
    psd::TopkSelectArgs s;
    memset(&s, 0, sizeof s);
    s.V = p->vocab;
    s.top_k = p->top_k;
    s.top_p = p->top_p;
    s.cap = p->top_k;
    s.list_tok = (int32_t*)(ws + T.tok);
    s.list_val = (float*)(ws + T.val);
    s.list_len = (int32_t*)(ws + T.len);
    s.list_lse = (float*)(ws + T.lse);
    s.radix_rows = (uint32_t*)(ws + L.ctrl) + psd::kCtrlTopkRadix;
    int ns = 0;
    if (draft_logits && s_count > 0) {
        psd::TopkSegment& g = s.seg[ns++];
        g.logits = draft_logits;
        g.n_rows = B * K * s_count;
        g.T = p->temp_draft;
        g.row_id_base = s_begin;
        g.group = s_count;
        g.group_stride = G;
        g.lse_out = draft_lse;
        g.lse_index_base = s_begin;
        g.lse_group_stride = G;
    }
    if (target_rows > 0) {
        psd::TopkSegment& g = s.seg[ns++];
        g.logits = target_logits;
        g.n_rows = B * target_rows * (G + 1);
        g.T = p->temp_target;
        g.row_id_base = B * K * G;
        g.lse_out = target_lse;
    }
    hipError_t e;
    if ((e = psd::launch_topk_select(s, bf16, stream)) != hipSuccess) return hip_fail(e, "top-k select launch");
    psd::TopkRaceArgs r;
    memset(&r, 0, sizeof r);
    r.prefix = b->prefix_tokens;
    r.start_pos = b->start_pos;
    r.draft_tokens = draft_tokens;
    r.out_tokens = out_tokens;
    r.out_len = out_len;
    r.target_tokens = target_tokens;
    r.list_tok = s.list_tok;
    r.list_val = s.list_val;
    r.list_len = s.list_len;
    r.cap = p->top_k;
    r.key = p->key;
    r.V = p->vocab;
    r.K = K;
    r.m = p->ctx_window;
    r.B = B;
    r.gamma = G;
    r.s_begin = s_begin;
    r.s_count = draft_logits ? s_count : 0;
    r.target_rows = target_rows;
    r.mpfr = p->mode == PSD_MODE_MPFR;
    r.T_target = p->temp_target;
    r.T_draft = p->temp_draft;
    r.chain = (int32_t*)(ws + T.chain);
    r.ctrl = (uint32_t*)(ws + L.ctrl);
    r.status = b->status;
    if ((e = psd::launch_topk_race(r, p->clocks, stream)) != hipSuccess) return hip_fail(e, "top-k race launch");
    return PSD_OK;
}

psd_status run_race(const psd_params* p, psd::RaceArgs& a, hipStream_t stream) {
    const size_t es = p->dtype == PSD_BF16 ? 2 : 4;
    bool vec = ((size_t)p->vocab * es) % 16 == 0;
    if (a.draft_logits) vec = vec && aligned16(a.draft_logits);
    if (a.target_logits) vec = vec && aligned16(a.target_logits);
    hipError_t e = psd::launch_race(a, p->dtype == PSD_BF16, vec, p->clocks, stream);
    if (e != hipSuccess) return hip_fail(e, "race kernel launch");
    return PSD_OK;
}

}  // namespace

extern "C" {

int32_t psd_abi_version(void) { return PSD_ABI_VERSION; }

const char* psd_last_error(void) { return g_err; }

void psd_set_spin_limit(uint32_t polls) { g_spin_limit.store(polls ? polls : kDefaultSpinLimit, std::memory_order_relaxed); }

size_t psd_workspace_bytes(const psd_params* params, int32_t batch, int32_t gamma) {
    if (!params || params->vocab < 1 || params->vocab > PSD_MAX_VOCAB || params->num_drafts < 1 ||
        params->num_drafts > PSD_MAX_DRAFTS || batch < 1 || gamma < 1 || gamma > PSD_MAX_GAMMA ||
        (params->dtype != PSD_F32 && params->dtype != PSD_BF16))
        return 0;
    if (params->top_k < 0 || params->top_k > PSD_MAX_TOP_K) return 0;
    return workspace_need(params, batch, gamma);
}

psd_status psd_workspace_clear(void* workspace, size_t workspace_bytes, hipStream_t stream) {
    if (!workspace) return fail(PSD_E_ARG, "workspace is NULL");
    if (((uintptr_t)workspace & 255u) != 0) return fail(PSD_E_WORKSPACE, "workspace must be 256-byte aligned");
    // The control region starts the workspace; clearing everything below the token slots of the
    // largest layout that fits is enough, but clearing the whole buffer is simplest and cheap.
    hipError_t e = psd::launch_fill_zero((uint32_t*)workspace, workspace_bytes / 4, stream);
    if (e != hipSuccess) return hip_fail(e, "workspace clear");
    return PSD_OK;
}

psd_status psd_workspace_errors(const void* workspace, hipStream_t stream, uint32_t* out_bits) {
    if (!workspace || !out_bits) return fail(PSD_E_ARG, "NULL argument");
    uint32_t ctrl[16];
    hipError_t e = hipMemcpyAsync(ctrl, workspace, sizeof ctrl, hipMemcpyDeviceToHost, stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    if (e != hipSuccess) return hip_fail(e, "workspace error read");
    *out_bits = ctrl[2];
    return PSD_OK;
}

psd_status psd_draft(const psd_params* params, const psd_block* block, int32_t s_begin, int32_t s_count,
                     const void* draft_logits, int32_t* draft_tokens, float* draft_lse, hipStream_t stream) {
    psd_status st = check_params(params);
    if (st != PSD_OK) return st;
    if ((st = check_block(params, block)) != PSD_OK) return st;
    if (s_begin < 0 || s_count < 1 || s_begin + s_count > block->gamma)
        return fail(PSD_E_ARG, "draft depths [%d, %d) outside [0, gamma=%d)", s_begin, s_begin + s_count, block->gamma);
    if (!draft_logits) return fail(PSD_E_ARG, "draft_logits is NULL");
    if (!draft_tokens) return fail(PSD_E_ARG, "draft_tokens is NULL");
    if (params->top_k > 0)
        return run_topk(params, block, s_begin, s_count, 0, nullptr, draft_logits, draft_tokens, nullptr, nullptr,
                        nullptr, draft_lse, nullptr, stream);
    if (params->mode == PSD_MODE_MPFR) {
        if ((st = run_mpfr_drafts(params, block, s_begin, s_count, draft_logits, draft_tokens, draft_lse, stream)) != PSD_OK)
            return st;
        const psd::WsLayout L = psd::ws_layout(block->batch, params->num_drafts, block->gamma, params->vocab,
                                               params->dtype == PSD_BF16);
        hipError_t e = psd::launch_finish_status((uint32_t*)((unsigned char*)block->workspace + L.ctrl), block->status, stream);
        if (e != hipSuccess) return hip_fail(e, "status kernel launch");
        return PSD_OK;
    }
    psd::RaceArgs a = base_args(params, block);
    a.draft_logits = draft_logits;
    a.draft_tokens = draft_tokens;
    a.draft_lse = draft_lse;
    a.s_begin = s_begin;
    a.s_count = s_count;
    a.target_rows = 0;
    build_depths(a, s_begin + s_count);
    return run_race(params, a, stream);
}

}  // extern "C"

namespace {

// Identical drafters with one shared target chain: the target chain needs no draft
// until the walk, so the fused kernel races it (without the walk) on the side
// stream while the drafts are sampled on the caller's stream (the draft rows are
// streamed on whichever stream lets the sampling start soonest); the walk kernel
// follows both.  The race kernel's error bits go to a control word that the walk
// kernel adds to the call's status.
psd_status verify_mpfr_forked(const psd_params* params, const psd_block* block, const void* target_logits,
                              const void* draft_logits, int32_t* draft_tokens, int32_t* out_tokens,
                              int32_t* out_len, float* target_lse, float* draft_lse, int32_t* target_tokens,
                              hipStream_t stream, Fork& f) {
    unsigned char* ws = (unsigned char*)block->workspace;
    const psd::WsLayout L = psd::ws_layout(block->batch, params->num_drafts, block->gamma, params->vocab,
                                           params->dtype == PSD_BF16);
    const psd::MpfrLayout M = psd::mpfr_layout(L, block->batch, params->num_drafts, block->gamma);
    uint32_t* ctrl = (uint32_t*)(ws + L.ctrl);
    int32_t* y = target_tokens ? target_tokens : (int32_t*)(ws + M.ytok);
    psd::RaceArgs a = base_args(params, block);
    a.target_logits = target_logits;
    a.draft_tokens = draft_tokens;
    a.out_tokens = out_tokens;
    a.out_len = out_len;
    a.target_lse = target_lse;
    a.target_tokens = y;
    a.s_begin = 0;
    a.s_count = 0;
    a.target_rows = 1;
    build_depths(a, block->gamma + 1);
    a.walk_kind = -1;  // no row walks: the walk kernel does, after the drafts
    a.status = ctrl + psd::kCtrlRaceBits;
    psd::MpfrArgs m = mpfr_args(params, block, 0, block->gamma, draft_logits, draft_tokens, draft_lse);
    bool streamed = false;
    psd_status st = mpfr_prepare(params, block, m, &streamed);
    if (st != PSD_OK) return st;
    hipError_t e;
    psd_status sd;
    if (streamed && m.tok_slot) {
        // One sampling launch for every depth on the caller's stream, which waits for
        // the streamed rows' tagged words, beside the streaming launch and then the
        // target race on the side stream (the streaming launch never waits, and both
        // launches' workgroups fit the device together).  The streaming launch is
        // enqueued first, so a sampling launch never waits for rows that will not come.
        // Half as many streaming workgroups as rows (two rows each, depth-major; at least
        // 512 or every row) land the first depths' rows sooner: 178 vs 185 us per call
        // with one per row at V=128256, K=4, gamma=4, B=64 (384: 191 us, 256: 209 us).
        const int rows = m.B * m.K * m.s_count;
        m.stream_grid = std::max((rows + 1) / 2, std::min(rows, 512));
        if ((e = hipEventRecord(f.in, stream)) != hipSuccess) return hip_fail(e, "fork event record");
        if ((e = hipStreamWaitEvent(f.side, f.in, 0)) != hipSuccess) return hip_fail(e, "fork event wait");
        if ((st = mpfr_stream_rows(params, m, f.side)) != PSD_OK) return st;
        // from here on the join is always enqueued, so the caller's stream never runs
        // ahead of the side stream
        sd = mpfr_sample_depths(params, m, stream);
        if (sd == PSD_OK) sd = run_race(params, a, f.side);
    } else {
        // The streaming pass (when there is one) first, on the caller's stream: the race
        // kernel, whose streaming workgroups would otherwise hold the device while it
        // runs, then overlaps only the depth launches (236 vs 256 us per call at
        // V=128256, K=4, gamma=4, B=64 with one launch per depth).
        if (streamed && (st = mpfr_stream_rows(params, m, stream)) != PSD_OK) return st;
        if ((e = hipEventRecord(f.in, stream)) != hipSuccess) return hip_fail(e, "fork event record");
        if ((e = hipStreamWaitEvent(f.side, f.in, 0)) != hipSuccess) return hip_fail(e, "fork event wait");
        if ((st = run_race(params, a, f.side)) != PSD_OK) return st;
        // from here on the join is always enqueued, so the caller's stream never runs
        // ahead of the side stream's race
        sd = mpfr_sample_depths(params, m, stream);
    }
    if ((e = hipEventRecord(f.out, f.side)) != hipSuccess) return hip_fail(e, "join event record");
    if ((e = hipStreamWaitEvent(stream, f.out, 0)) != hipSuccess) return hip_fail(e, "join event wait");
    if (sd != PSD_OK) return sd;
    psd::TopkRaceArgs w;
    memset(&w, 0, sizeof w);
    w.draft_tokens = draft_tokens;
    w.out_tokens = out_tokens;
    w.out_len = out_len;
    w.chain = y;
    w.K = params->num_drafts;
    w.B = block->batch;
    w.gamma = block->gamma;
    w.ctrl = ctrl;
    w.status = block->status;
    w.status_in = ctrl + psd::kCtrlRaceBits;
    if ((e = psd::launch_walk(w, stream)) != hipSuccess) return hip_fail(e, "walk kernel launch");
    return PSD_OK;
}

// may_fork: the identical-drafter form may use the side stream (not under stream
// capture, and not from the allocation-free entry point).
psd_status verify_impl(const psd_params* params, const psd_block* block, int32_t target_rows,
                       const void* target_logits, const void* draft_logits, int32_t* draft_tokens,
                       int32_t* out_tokens, int32_t* out_len, float* target_lse, float* draft_lse,
                       int32_t* target_tokens, hipStream_t stream, bool may_fork) {
    psd_status st;
    if ((st = check_block(params, block)) != PSD_OK) return st;
    if (target_rows != 1 && target_rows != params->num_drafts)
        return fail(PSD_E_ARG, "target_rows must be 1 or num_drafts (%d), got %d", params->num_drafts, target_rows);
    if (!target_logits) return fail(PSD_E_ARG, "target_logits is NULL");
    if (!draft_tokens) return fail(PSD_E_ARG, "draft_tokens is NULL");
    if (!out_tokens || !out_len) return fail(PSD_E_ARG, "out_tokens / out_len is NULL");
    if (!draft_logits && draft_lse) return fail(PSD_E_ARG, "draft_lse requires draft_logits");
    if (params->top_k > 0)
        return run_topk(params, block, 0, block->gamma, target_rows, target_logits, draft_logits, draft_tokens,
                        out_tokens, out_len, target_lse, draft_lse, target_tokens, stream);
    if (params->mode == PSD_MODE_MPFR && draft_logits && target_rows == 1 && may_fork) {
        hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
        hipError_t e = hipStreamIsCapturing(stream, &cs);
        if (e != hipSuccess) return hip_fail(e, "stream capture query");
        if (cs == hipStreamCaptureStatusNone) {
            std::lock_guard<std::mutex> lock(g_fork_mu);
            Fork* f = fork_objects();
            if (f)
                return verify_mpfr_forked(params, block, target_logits, draft_logits, draft_tokens, out_tokens,
                                          out_len, target_lse, draft_lse, target_tokens, stream, *f);
        }
    }
    if (params->mode == PSD_MODE_MPFR && draft_logits) {
        // identical drafters: the context tree is drafted depth by depth first, then the
        // target rows race slot 0 in the fused kernel with the drafts as input
        if ((st = run_mpfr_drafts(params, block, 0, block->gamma, draft_logits, draft_tokens, draft_lse, stream)) != PSD_OK)
            return st;
        draft_logits = nullptr;
        draft_lse = nullptr;
    }
    psd::RaceArgs a = base_args(params, block);
    a.target_logits = target_logits;
    a.draft_logits = draft_logits;
    a.draft_tokens = draft_tokens;
    a.out_tokens = out_tokens;
    a.out_len = out_len;
    a.target_lse = target_lse;
    a.draft_lse = draft_lse;
    a.target_tokens = target_tokens;
    a.s_begin = 0;
    a.s_count = draft_logits ? block->gamma : 0;
    a.target_rows = target_rows;
    build_depths(a, block->gamma + 1);
    return run_race(params, a, stream);
}

}  // namespace

extern "C" {

psd_status psd_verify(const psd_params* params, const psd_block* block, int32_t target_rows,
                      const void* target_logits, const void* draft_logits, int32_t* draft_tokens,
                      int32_t* out_tokens, int32_t* out_len, float* target_lse, float* draft_lse,
                      int32_t* target_tokens, hipStream_t stream) {
    psd_status st = check_params(params);
    if (st != PSD_OK) return st;
    return verify_impl(params, block, target_rows, target_logits, draft_logits, draft_tokens, out_tokens, out_len,
                       target_lse, draft_lse, target_tokens, stream, true);
}

psd_status psd_verify_static(const psd_params* params, const psd_block* block, int32_t target_rows,
                             const void* target_logits, const void* draft_logits, int32_t* draft_tokens,
                             int32_t* out_tokens, int32_t* out_len, float* target_lse, float* draft_lse,
                             int32_t* target_tokens, hipStream_t stream) {
    psd_status st = check_params(params);
    if (st != PSD_OK) return st;
    if (!block) return fail(PSD_E_ARG, "block is NULL");
    if (block->workspace || block->workspace_bytes)
        return fail(PSD_E_ARG, "psd_verify_static uses the library's fixed scratch: pass workspace NULL, 0 bytes");
    if (block->batch < 1 || block->gamma < 1 || block->gamma > PSD_MAX_GAMMA)
        return fail(PSD_E_ARG, "batch %d / gamma %d out of range", block->batch, block->gamma);
    const size_t need = workspace_need(params, block->batch, block->gamma);
    if (need > psd::kStaticScratchBytes)
        return fail(PSD_E_WORKSPACE, "the shape needs %zu bytes of scratch; the fixed scratch holds %zu "
                    "(use psd_verify with a workspace)", need, psd::kStaticScratchBytes);
    void* ws = nullptr;
    hipError_t e = psd::static_scratch(&ws, stream);
    if (e != hipSuccess) return hip_fail(e, "fixed scratch");
    psd_block b = *block;
    b.workspace = ws;
    b.workspace_bytes = psd::kStaticScratchBytes;
    return verify_impl(params, &b, target_rows, target_logits, draft_logits, draft_tokens, out_tokens, out_len,
                       target_lse, draft_lse, target_tokens, stream, false);
}

psd_status psd_detect(const psd_params* params, int32_t n_seq, int32_t seq_len, const int32_t* tokens,
                      const int32_t* n0, double* out_score, int32_t* out_count, float* out_per_token,
                      hipStream_t stream) {
    psd_status st = check_params(params);
    if (st != PSD_OK) return st;
    if (n_seq < 0 || seq_len < 0) return fail(PSD_E_ARG, "negative n_seq / seq_len");
    if (n_seq > 0 && (!tokens || !n0 || !out_score || !out_count))
        return fail(PSD_E_ARG, "tokens / n0 / out_score / out_count is NULL");
    psd::DetectArgs a;
    memset(&a, 0, sizeof a);
    a.row_stride = seq_len;
    a.tokens = tokens;
    a.n0 = n0;
    a.out_score = out_score;
    a.out_count = out_count;
    a.out_per_token = out_per_token;
    a.key = params->key;
    a.n_seq = n_seq;
    a.seq_len = seq_len;
    a.V = params->vocab;
    // identical drafters: the target races slot 0 alone, whose clock is the pivot (K = 1)
    a.K = params->mode == PSD_MODE_MPFR ? 1 : params->num_drafts;
    a.m = params->ctx_window;
    hipError_t e = psd::launch_detect(a, params->clocks, stream);
    if (e != hipSuccess) return hip_fail(e, "detect kernel launch");
    return PSD_OK;
}

}  // extern "C"

namespace {

// Li et al.'s k_Delta, q_Delta: 1/(1 - Delta) within 1e-12 (relative) of an integer counts
// as that integer, and then q = 0 (binary rounding must not leave q ~ 1e-16).
psd_status score_params(const psd_score_params* sp, double& lnk, double& a, double& b, int& qpos, double& cap,
                        double& c0) {
    if (!sp) return fail(PSD_E_ARG, "score params is NULL");
    if (!(sp->li_delta > 0.0 && sp->li_delta < 1.0)) return fail(PSD_E_ARG, "li_delta must be in (0, 1)");
    if (!(sp->pl_eps > 0.0 && sp->pl_eps <= 1.0)) return fail(PSD_E_ARG, "pl_eps must be in (0, 1]");
    const double d = sp->li_delta, x = 1.0 / (1.0 - d);
    const double k = floor(x + 1e-12 * x);
    double q = 1.0 - k * (1.0 - d);
    if (q < 1e-12) q = 0.0;
    lnk = log(k);
    a = d / (1.0 - d);
    b = q > 0.0 ? (1.0 - q) / q : 0.0;
    qpos = q > 0.0;
    cap = 1.0 / sqrt(sp->pl_eps);
    c0 = 2.0 - sqrt(sp->pl_eps);
    return PSD_OK;
}

}  // namespace

extern "C" {

psd_status psd_detect_scores(const psd_params* params, const psd_score_params* sp, int32_t n_seq, int32_t seq_len,
                             int32_t row_stride, const int32_t* tokens, const int32_t* n0, double* out_scores,
                             int32_t* out_count, hipStream_t stream) {
    psd_status st = check_params(params);
    if (st != PSD_OK) return st;
    if (n_seq < 0 || seq_len < 0) return fail(PSD_E_ARG, "negative n_seq / seq_len");
    if (row_stride < seq_len) return fail(PSD_E_ARG, "row_stride %d < seq_len %d", row_stride, seq_len);
    if (n_seq > 0 && (!tokens || !n0 || !out_scores || !out_count))
        return fail(PSD_E_ARG, "tokens / n0 / out_scores / out_count is NULL");
    psd::DetectArgs a;
    memset(&a, 0, sizeof a);
    if ((st = score_params(sp, a.li_lnk, a.li_a, a.li_b, a.li_q, a.pl_cap, a.pl_c0)) != PSD_OK) return st;
    a.tokens = tokens;
    a.n0 = n0;
    a.out_score = out_scores;
    a.out_count = out_count;
    a.key = params->key;
    a.n_seq = n_seq;
    a.seq_len = seq_len;
    a.row_stride = row_stride;
    a.V = params->vocab;
    a.K = params->mode == PSD_MODE_MPFR ? 1 : params->num_drafts;
    a.m = params->ctx_window;
    a.multi = 1;
    hipError_t e = psd::launch_detect(a, params->clocks, stream);
    if (e != hipSuccess) return hip_fail(e, "detect kernel launch");
    return PSD_OK;
}

psd_status psd_detect_scores_pvalue(const psd_score_params* sp, int32_t n_seq, const double* scores,
                                    const int32_t* count, double* out_log_p, hipStream_t stream) {
    psd::ScorePvalueArgs a;
    memset(&a, 0, sizeof a);
    psd_status st = score_params(sp, a.li_lnk, a.li_a, a.li_b, a.li_q, a.pl_cap, a.pl_c0);
    if (st != PSD_OK) return st;
    if (n_seq < 0) return fail(PSD_E_ARG, "n_seq < 0");
    if (n_seq > 0 && (!scores || !count || !out_log_p)) return fail(PSD_E_ARG, "scores / count / out_log_p is NULL");
    a.scores = scores;
    a.count = count;
    a.out_log_p = out_log_p;
    a.n = n_seq;
    a.pl_eps = sp->pl_eps;
    hipError_t e = psd::launch_score_pvalues(a, stream);
    if (e != hipSuccess) return hip_fail(e, "score p-value kernel launch");
    return PSD_OK;
}

psd_status psd_detection_rate(int32_t n, const double* log_p, int32_t stride, double alpha, int32_t* out_count,
                              hipStream_t stream) {
    if (n < 0 || stride < 1) return fail(PSD_E_ARG, "n < 0 or stride < 1");
    if (!(alpha > 0.0 && alpha <= 1.0)) return fail(PSD_E_ARG, "alpha must be in (0, 1]");
    if (!out_count || (n > 0 && !log_p)) return fail(PSD_E_ARG, "log_p / out_count is NULL");
    hipError_t e = psd::launch_detection_rate(n, log_p, stride, log(alpha), out_count, stream);
    if (e != hipSuccess) return hip_fail(e, "detection rate kernel launch");
    return PSD_OK;
}

psd_status psd_detect_pvalue(int32_t n_seq, const double* score, const int32_t* count, double* out_log_p,
                             double* out_anlppt, hipStream_t stream) {
    if (n_seq < 0) return fail(PSD_E_ARG, "n_seq < 0");
    if (n_seq > 0 && (!score || !count || !out_log_p)) return fail(PSD_E_ARG, "score / count / out_log_p is NULL");
    hipError_t e = psd::launch_pvalue(n_seq, score, count, out_log_p, out_anlppt, stream);
    if (e != hipSuccess) return hip_fail(e, "p-value kernel launch");
    return PSD_OK;
}

psd_status psd_philox(int32_t n, const uint32_t* ctr, const uint32_t* key, uint32_t* out, hipStream_t stream) {
    if (n < 0) return fail(PSD_E_ARG, "n < 0");
    if (n > 0 && (!ctr || !key || !out)) return fail(PSD_E_ARG, "NULL argument");
    hipError_t e = psd::launch_philox(n, ctr, key, out, stream);
    if (e != hipSuccess) return hip_fail(e, "philox kernel launch");
    return PSD_OK;
}

psd_status psd_context_keys(const psd_params* params, int32_t n, const int64_t* t, const int32_t* windows,
                            uint32_t* out_kappa, hipStream_t stream) {
    if (!params) return fail(PSD_E_ARG, "params is NULL");
    if (params->ctx_window < 0 || params->ctx_window > PSD_MAX_WINDOW) return fail(PSD_E_ARG, "bad ctx_window");
    if (n < 0) return fail(PSD_E_ARG, "n < 0");
    if (n > 0 && (!t || !out_kappa || (params->ctx_window > 0 && !windows))) return fail(PSD_E_ARG, "NULL argument");
    hipError_t e = psd::launch_context_keys(params->key, params->ctx_window, n, t, windows, out_kappa, stream);
    if (e != hipSuccess) return hip_fail(e, "context key kernel launch");
    return PSD_OK;
}

psd_status psd_clock_values(const psd_params* params, int32_t n, const uint32_t* kappa, const int32_t* slot,
                            const int32_t* token, double* out, hipStream_t stream) {
    if (!params) return fail(PSD_E_ARG, "params is NULL");
    if (params->vocab < 1 || params->vocab > PSD_MAX_VOCAB) return fail(PSD_E_ARG, "bad vocab");
    if (params->clocks != PSD_CLOCKS_TREE && params->clocks != PSD_CLOCKS_FLAT) return fail(PSD_E_ARG, "bad clocks");
    if (n < 0) return fail(PSD_E_ARG, "n < 0");
    if (n > 0 && (!kappa || !slot || !token || !out)) return fail(PSD_E_ARG, "NULL argument");
    hipError_t e = psd::launch_clock_values(params->clocks, params->vocab, n, kappa, slot, token, out, stream);
    if (e != hipSuccess) return hip_fail(e, "clock kernel launch");
    return PSD_OK;
}

}  // extern "C"

// ---------------------------------------------------------------- multi-block generation

namespace {

// psd_generate's scratch: the block workspace first (so it keeps its alignment),
// then both logits buffers and the loop's state.
struct GenLayout {
    size_t ws_bytes, tl, dl, dt, ot, ol, len, start, prefix, active, total;
};

GenLayout gen_layout(const psd_params* p, int B, int G) {
    GenLayout L;
    const size_t es = p->dtype == PSD_BF16 ? 2 : 4, V = (size_t)p->vocab, K = (size_t)p->num_drafts;
    L.ws_bytes = workspace_need(p, B, G);
    size_t o = psd::align256(L.ws_bytes);
    L.tl = o;
    o = psd::align256(o + (size_t)B * (G + 1) * V * es);
    L.dl = o;
    o = psd::align256(o + (size_t)B * K * G * V * es);
    L.dt = o;
    o = psd::align256(o + (size_t)B * K * G * 4);
    L.ot = o;
    o = psd::align256(o + (size_t)B * (G + 1) * 4);
    L.ol = o;
    o = psd::align256(o + (size_t)B * 4);
    L.len = o;
    o = psd::align256(o + (size_t)B * 8);
    L.start = o;
    o = psd::align256(o + (size_t)B * 8);
    L.prefix = o;
    o = psd::align256(o + (size_t)B * (size_t)p->ctx_window * 4 + 4);
    L.active = o;
    o = psd::align256(o + 4);
    L.total = o;
    return L;
}

psd_status check_toy(const psd_toy_lm* lm) {
    if (!lm) return fail(PSD_E_ARG, "toy model is NULL");
    if (!isfinite(lm->sigma) || !isfinite(lm->alpha) || !isfinite(lm->tau[0]) || !isfinite(lm->tau[1]))
        return fail(PSD_E_ARG, "toy model parameters must be finite");
    return PSD_OK;
}

psd::ToyArgs toy_args(const psd_params* p, const psd_toy_lm* lm, int B, int G, const int64_t* start, void* tl,
                      void* dl) {
    psd::ToyArgs a;
    memset(&a, 0, sizeof a);
    a.start_pos = start;
    a.target_logits = tl;
    a.draft_logits = dl;
    a.seed = lm->seed;
    a.draft_seed = lm->draft_seed;
    a.sigma = lm->sigma;
    a.w = (float)(-(double)lm->alpha * 0.69314718055994531 * 0x1p-23);
    a.tau0 = lm->tau[0];
    a.tau1 = lm->tau[1];
    a.tau_split = lm->tau_split;
    a.V = p->vocab;
    a.K = p->num_drafts;
    a.B = B;
    a.gamma = G;
    return a;
}

psd::AdvanceArgs advance_args(int B, int G, int m, int64_t max_len, const int32_t* out_tokens, const int32_t* out_len,
                              int32_t* text, int64_t text_stride, int64_t* length, int32_t* prefix, int64_t* start,
                              int32_t* n_active) {
    psd::AdvanceArgs a;
    memset(&a, 0, sizeof a);
    a.out_tokens = out_tokens;
    a.out_len = out_len;
    a.text = text;
    a.text_stride = text_stride;
    a.length = length;
    a.start_pos = start;
    a.prefix = prefix;
    a.n_active = n_active;
    a.B = B;
    a.gamma = G;
    a.m = m;
    a.max_len = max_len;
    return a;
}

psd_status check_shape(int32_t batch, int32_t gamma) {
    if (batch < 1 || batch > PSD_MAX_BATCH) return fail(PSD_E_ARG, "batch %d outside [1, %d]", batch, PSD_MAX_BATCH);
    if (gamma < 1 || gamma > PSD_MAX_GAMMA) return fail(PSD_E_ARG, "gamma %d outside [1, %d]", gamma, PSD_MAX_GAMMA);
    return PSD_OK;
}

}  // namespace

extern "C" {

psd_status psd_advance(const psd_params* params, int32_t batch, int32_t gamma, int64_t max_len,
                       const int32_t* out_tokens, const int32_t* out_len, int32_t* text, int64_t text_stride,
                       int64_t* length, int32_t* prefix_tokens, int64_t* start_pos, int32_t* n_active,
                       hipStream_t stream) {
    if (!params) return fail(PSD_E_ARG, "params is NULL");
    const int m = params->ctx_window;
    if (m < 0 || m > PSD_MAX_WINDOW) return fail(PSD_E_ARG, "ctx_window %d outside [0, %d]", m, PSD_MAX_WINDOW);
    psd_status st = check_shape(batch, gamma);
    if (st != PSD_OK) return st;
    if (max_len <= m) return fail(PSD_E_ARG, "max_len must exceed the prompt length m = %d", m);
    if (text_stride < max_len) return fail(PSD_E_ARG, "text_stride is below max_len");
    if (!text || !length || !start_pos || !n_active || (m > 0 && !prefix_tokens))
        return fail(PSD_E_ARG, "text / length / start_pos / n_active / prefix_tokens is NULL");
    if (out_len && !out_tokens) return fail(PSD_E_ARG, "out_tokens is NULL");
    hipError_t e = psd::launch_advance(advance_args(batch, gamma, m, max_len, out_tokens, out_len, text, text_stride,
                                                    length, prefix_tokens, start_pos, n_active),
                                       stream);
    if (e != hipSuccess) return hip_fail(e, "advance kernel launch");
    return PSD_OK;
}

psd_status psd_toy_logits(const psd_params* params, const psd_toy_lm* lm, int32_t batch, int32_t gamma,
                          const int64_t* start_pos, void* target_logits, void* draft_logits, hipStream_t stream) {
    psd_status st = check_params(params);
    if (st != PSD_OK) return st;
    if ((st = check_toy(lm)) != PSD_OK) return st;
    if ((st = check_shape(batch, gamma)) != PSD_OK) return st;
    if (!start_pos || !target_logits) return fail(PSD_E_ARG, "start_pos / target_logits is NULL");
    hipError_t e = psd::launch_toy_rows(toy_args(params, lm, batch, gamma, start_pos, target_logits, draft_logits),
                                        params->dtype == PSD_BF16, stream);
    if (e != hipSuccess) return hip_fail(e, "toy model kernel launch");
    return PSD_OK;
}

size_t psd_generate_workspace_bytes(const psd_params* params, int32_t batch, int32_t gamma) {
    if (psd_workspace_bytes(params, batch, gamma) == 0) return 0;
    if (params->ctx_window < 0 || params->ctx_window > PSD_MAX_WINDOW) return 0;
    return gen_layout(params, batch, gamma).total;
}

psd_status psd_generate(const psd_params* params, const psd_toy_lm* lm, int32_t batch, int32_t gamma, int32_t n_pos,
                        int32_t* text, int64_t text_stride, void* workspace, size_t workspace_bytes,
                        int32_t check_every, int32_t use_graph, int32_t* out_blocks, uint32_t* out_status,
                        hipStream_t stream) {
    psd_status st = check_params(params);
    if (st != PSD_OK) return st;
    if ((st = check_toy(lm)) != PSD_OK) return st;
    if ((st = check_shape(batch, gamma)) != PSD_OK) return st;
    const int m = params->ctx_window;
    if (n_pos < 1) return fail(PSD_E_ARG, "n_pos must be at least 1");
    if (!text) return fail(PSD_E_ARG, "text is NULL");
    if (text_stride < (int64_t)m + n_pos) return fail(PSD_E_ARG, "text_stride is below m + n_pos");
    if (check_every < 1) return fail(PSD_E_ARG, "check_every must be at least 1");
    const GenLayout L = gen_layout(params, batch, gamma);
    if (!workspace) return fail(PSD_E_WORKSPACE, "workspace is NULL");
    if (((uintptr_t)workspace & 255u) != 0) return fail(PSD_E_WORKSPACE, "workspace must be 256-byte aligned");
    if (workspace_bytes < L.total)
        return fail(PSD_E_WORKSPACE, "workspace has %zu bytes, needs %zu", workspace_bytes, L.total);
    unsigned char* ws = (unsigned char*)workspace;
    const int64_t max_len = (int64_t)m + n_pos;
    const bool bf16 = params->dtype == PSD_BF16;
    void* tl = ws + L.tl;
    void* dl = ws + L.dl;
    int32_t* dt = (int32_t*)(ws + L.dt);
    int32_t* ot = (int32_t*)(ws + L.ot);
    int32_t* ol = (int32_t*)(ws + L.ol);
    int64_t* len = (int64_t*)(ws + L.len);
    int64_t* start = (int64_t*)(ws + L.start);
    int32_t* prefix = (int32_t*)(ws + L.prefix);
    int32_t* active = (int32_t*)(ws + L.active);
    psd_block blk;
    memset(&blk, 0, sizeof blk);
    blk.batch = batch;
    blk.gamma = gamma;
    blk.prefix_tokens = prefix;
    blk.start_pos = start;
    blk.workspace = ws;
    blk.workspace_bytes = L.ws_bytes;
    const psd::ToyArgs toy = toy_args(params, lm, batch, gamma, start, tl, dl);
    const psd::AdvanceArgs adv = advance_args(batch, gamma, m, max_len, ot, ol, text, text_stride, len, prefix, start,
                                              active);
    // one block: the model's rows, the race and the walk, the commit
    auto body = [&](hipStream_t s) -> psd_status {
        hipError_t e = psd::launch_toy_rows(toy, bf16, s);
        if (e != hipSuccess) return hip_fail(e, "toy model kernel launch");
        psd_status r = verify_impl(params, &blk, 1, tl, dl, dt, ot, ol, nullptr, nullptr, nullptr, s, false);
        if (r != PSD_OK) return r;
        if ((e = psd::launch_advance(adv, s)) != hipSuccess) return hip_fail(e, "advance kernel launch");
        return PSD_OK;
    };

    hipStream_t s = stream, own = nullptr;
    hipEvent_t ev = nullptr;
    hipGraph_t graph = nullptr;
    hipGraphExec_t exec = nullptr;
    int32_t* host_active = nullptr;
    int blocks = 0;
    hipError_t e = hipSuccess;
    st = PSD_OK;
    do {
        if (use_graph) {
            // capture needs a stream of its own (the caller's may be the null stream)
            if ((e = hipStreamCreateWithFlags(&own, hipStreamNonBlocking)) != hipSuccess) break;
            if ((e = hipEventCreateWithFlags(&ev, hipEventDisableTiming)) != hipSuccess) break;
            if ((e = hipEventRecord(ev, stream)) != hipSuccess) break;
            if ((e = hipStreamWaitEvent(own, ev, 0)) != hipSuccess) break;
            s = own;
        }
        if ((e = hipHostMalloc((void**)&host_active, sizeof(int32_t), hipHostMallocDefault)) != hipSuccess) break;
        // a fresh block workspace, and the first block's windows from the prompts
        if ((e = psd::launch_fill_zero((uint32_t*)ws, L.ws_bytes / 4, s)) != hipSuccess) break;
        psd::AdvanceArgs first = adv;
        first.out_len = nullptr;
        if ((e = psd::launch_advance(first, s)) != hipSuccess) break;
        if (use_graph) {
            if ((e = hipStreamBeginCapture(s, hipStreamCaptureModeRelaxed)) != hipSuccess) break;
            for (int i = 0; i < check_every && st == PSD_OK; ++i) st = body(s);
            hipGraph_t g = nullptr;
            const hipError_t ec = hipStreamEndCapture(s, &g);
            graph = g;
            if (st != PSD_OK) break;
            if ((e = ec) != hipSuccess) break;
            if ((e = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0)) != hipSuccess) break;
        }
        // every active sequence gains at least one token per block, so n_pos blocks suffice
        while (true) {
            if (use_graph) {
                if ((e = hipGraphLaunch(exec, s)) != hipSuccess) break;
            } else {
                for (int i = 0; i < check_every && st == PSD_OK; ++i) st = body(s);
                if (st != PSD_OK) break;
            }
            blocks += check_every;
            if ((e = hipMemcpyAsync(host_active, active, sizeof(int32_t), hipMemcpyDeviceToHost, s)) != hipSuccess)
                break;
            if ((e = hipStreamSynchronize(s)) != hipSuccess) break;
            if (*host_active == 0) break;
            if (blocks >= n_pos + check_every) {
                st = fail(PSD_E_HIP, "generation did not finish within %d blocks", blocks);
                break;
            }
        }
    } while (false);
    if (e != hipSuccess && st == PSD_OK) st = hip_fail(e, "generation loop");
    if (own) hipStreamSynchronize(own);
    if (exec) hipGraphExecDestroy(exec);
    if (graph) hipGraphDestroy(graph);
    if (host_active) hipHostFree(host_active);
    if (ev) hipEventDestroy(ev);
    if (own) hipStreamDestroy(own);
    if (st != PSD_OK) return st;
    if (out_blocks) *out_blocks = blocks;
    if (out_status) {
        uint32_t bits = 0;
        if ((st = psd_workspace_errors(ws, stream, &bits)) != PSD_OK) return st;
        *out_status = bits;
    }
    return PSD_OK;
}

}  // extern "C"
