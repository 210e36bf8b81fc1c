/*
 * psd_oracle.c -- plain, slow CPU oracle of the keyed Poisson/exponential race
 * ("Watermarkable Multi-Draft Speculative Sampling via Poisson Processes").
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or call
 * this file: only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg
 * use it.  It shares no code, header, table or constant with the HIP library; the
 * constants below are written out here from the published definitions.
 *
 * Everything is double precision, plain loops, no blocking, no pruning: every
 * clock a race uses is materialised and the argmin is exhaustive.
 *
 * Paper passages followed (by section / equation / algorithm):
 *  - keyed source Pi(c) = G(k, Lambda(c)), independent across contexts, tokens and
 *    arrival indices: Sec. 4.3 (single-draft algorithm), Sec. 5 (multi-draft
 *    algorithm), App. "Algorithm Implementation" (labeler Lambda, detector).
 *  - EFR race  Z = argmin_z E_z / P(z), E_z iid Exp(1), E_z/P(z)=+inf if P(z)=0:
 *    eq. (EFR) and Thm. "PFR reduces to EFR" (App. on PFR in the discrete case).
 *  - non-identical proposals, augmented space V x [B]: target races
 *    P~(i,b)=p_i/B over all (i,b), draft b races its own block b:
 *    Prop. "heterogeneous PML bound" (App. "Extension ... non-identically
 *    distributed proposals").
 *  - detector score A_t = -log(1 - r_t(w_t)): eq. (S_A), Sec. 4.3 and App.
 *    "Gumbel Watermark".
 *
 * Readings taken where the paper is silent (the paper fixes no PRF, PRNG or
 * counter layout): Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11); context
 * label = (key, absolute position t, previous m tokens); uniforms
 * U = (2*(w>>9)+1)*2^-24; E = -ln U; scores in natural log; exact ties go to the
 * lowest token, then the lowest slot.
 *
 * Two clock layouts define the same law (iid Exp(1) per (slot, token)):
 *  FLAT (layout 1): E_j[v] = -ln U(Philox(ctr=(v>>2, j, 0, 0), kappa)[v & 3]).
 *  TREE (layout 0): a top-down construction of the same iid field.  Tokens are
 *    grouped in a fixed hierarchy (level 1 = 8 tokens, then 16-ary: 128, 2048,
 *    32768 tokens, level 5 = the whole vocabulary, V <= 2^19).  For iid Exp(1)
 *    variables the minimum of a node of n tokens is Exp(1)/n, its position is
 *    uniform, and every other token of the node exceeds the minimum by an
 *    independent Exp(1) (memorylessness).  Hence a node that does not hold its
 *    parent's minimum has minimum m_parent + E'/n at a uniform position, and a
 *    token that is not its chunk's minimum has clock m_chunk + E'.  Expanding
 *    this recursion everywhere yields iid Exp(1) clocks for every token (the
 *    exponential-race form of the top-down Gumbel-process construction of
 *    Maddison, Tarlow and Minka, "A* Sampling", NIPS 2014).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ---------------- Philox4x32-10 (Salmon et al., SC'11) ------------------- */

#define ORC_PHILOX_M0 0xD2511F53u
#define ORC_PHILOX_M1 0xCD9E8D57u
#define ORC_PHILOX_W0 0x9E3779B9u
#define ORC_PHILOX_W1 0xBB67AE85u

void oracle_philox(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
    uint32_t x0 = ctr[0], x1 = ctr[1], x2 = ctr[2], x3 = ctr[3];
    uint32_t k0 = key[0], k1 = key[1];
    for (int round = 0; round < 10; round++) {
        if (round > 0) {
            k0 += ORC_PHILOX_W0;
            k1 += ORC_PHILOX_W1;
        }
        uint64_t prod0 = (uint64_t)ORC_PHILOX_M0 * (uint64_t)x0;
        uint64_t prod1 = (uint64_t)ORC_PHILOX_M1 * (uint64_t)x2;
        uint32_t hi0 = (uint32_t)(prod0 >> 32), lo0 = (uint32_t)prod0;
        uint32_t hi1 = (uint32_t)(prod1 >> 32), lo1 = (uint32_t)prod1;
        uint32_t y0 = hi1 ^ x1 ^ k0;
        uint32_t y1 = lo1;
        uint32_t y2 = hi0 ^ x3 ^ k1;
        uint32_t y3 = lo0;
        x0 = y0; x1 = y1; x2 = y2; x3 = y3;
    }
    out[0] = x0; out[1] = x1; out[2] = x2; out[3] = x3;
}

/* ---------------- context label -> keyed source ------------------------- */

/* fold(kappa, a, b, tag) = words 0 and 1 of Philox(ctr=(a, b, tag, 1), kappa).
 * Counter word 3 = 1 marks the key-derivation domain (clock counters use 0 or 2). */
void oracle_fold(const uint32_t kin[2], uint32_t a, uint32_t b, uint32_t tag, uint32_t kout[2]) {
    uint32_t ctr[4] = {a, b, tag, 1u};
    uint32_t w[4];
    oracle_philox(ctr, kin, w);
    kout[0] = w[0];
    kout[1] = w[1];
}

/* kappa = H(key, t, w_{t-m..t-1}): the labeler of the keyed source.
 * window[] holds the m previous tokens oldest -> newest; a missing token
 * (text shorter than m) is -1, i.e. 0xFFFFFFFF. */
void oracle_context_key(uint64_t key, int64_t t, const int32_t *window, int m, uint32_t kappa[2]) {
    uint32_t k[2] = {(uint32_t)key, (uint32_t)(key >> 32)};
    uint64_t tu = (uint64_t)t;
    uint32_t cur[2];
    oracle_fold(k, (uint32_t)tu, (uint32_t)(tu >> 32), 0u, cur);
    for (int i = 0; i < m; i++) {
        uint32_t nxt[2];
        oracle_fold(cur, (uint32_t)window[i], (uint32_t)i, 1u, nxt);
        cur[0] = nxt[0];
        cur[1] = nxt[1];
    }
    kappa[0] = cur[0];
    kappa[1] = cur[1];
}

/* ---------------- uniforms and clocks ----------------------------------- */

/* U = (2*(w>>9)+1) * 2^-24: 2^23 odd multiples of 2^-24, strictly inside (0,1). */
double oracle_uniform(uint32_t w) {
    return (2.0 * (double)(w >> 9) + 1.0) * (1.0 / 16777216.0);
}

static double orc_exp1(uint32_t w) { return -log(oracle_uniform(w)); }

/* FLAT layout: one Philox word per (slot, token). */
static double orc_flat_clock(const uint32_t kappa[2], int slot, int v) {
    uint32_t ctr[4] = {(uint32_t)v >> 2, (uint32_t)slot, 0u, 0u};
    uint32_t w[4];
    oracle_philox(ctr, kappa, w);
    return orc_exp1(w[v & 3]);
}

/* TREE layout hierarchy: node (level L, index i) covers tokens
 * [i << SH[L], min((i+1) << SH[L], V)). */
static const int ORC_SH[6] = {0, 3, 7, 11, 15, 19};

/* Draw attached to node (L, i): E' = -ln U(w0), uniform position
 * P = floor(n * W / 2^64) with W = (w1 << 32) | w2  (exact integer arithmetic). */
static void orc_node_draw(const uint32_t kappa[2], int slot, int L, uint32_t i, uint32_t n,
                          double *eprime, uint32_t *pos) {
    uint32_t ctr[4] = {i, (uint32_t)slot, (uint32_t)L, 2u};
    uint32_t w[4];
    oracle_philox(ctr, kappa, w);
    *eprime = orc_exp1(w[0]);
    uint64_t t = (uint64_t)w[2] * (uint64_t)n;
    uint64_t u = (uint64_t)w[1] * (uint64_t)n + (t >> 32);
    *pos = (uint32_t)(u >> 32);
}

/* Token draw: word (v & 3) of Philox(ctr=(v>>3, slot, 8 + ((v>>2)&1), 2), kappa). */
static double orc_token_draw(const uint32_t kappa[2], int slot, uint32_t v) {
    uint32_t ctr[4] = {v >> 3, (uint32_t)slot, 8u + ((v >> 2) & 1u), 2u};
    uint32_t w[4];
    oracle_philox(ctr, kappa, w);
    return orc_exp1(w[v & 3u]);
}

static uint32_t orc_node_start(int L, uint32_t i) { return i << ORC_SH[L]; }
static uint32_t orc_node_end(int L, uint32_t i, uint32_t V) {
    uint64_t e = ((uint64_t)i + 1u) << ORC_SH[L];
    return e < V ? (uint32_t)e : V;
}

/* Full expansion: node (L, i) has minimum m at token p; write every clock. */
static void orc_tree_expand(const uint32_t kappa[2], int slot, uint32_t V, int L, uint32_t i,
                            double m, uint32_t p, double *E) {
    uint32_t s = orc_node_start(L, i), e = orc_node_end(L, i, V);
    if (L == 1) {
        for (uint32_t v = s; v < e; v++)
            E[v] = (v == p) ? m : m + orc_token_draw(kappa, slot, v);
        return;
    }
    uint32_t c0 = s >> ORC_SH[L - 1];
    for (uint32_t c = c0;; c++) {
        uint32_t cs = orc_node_start(L - 1, c);
        if (cs >= e) break;
        uint32_t ce = orc_node_end(L - 1, c, V);
        if (p >= cs && p < ce) {
            orc_tree_expand(kappa, slot, V, L - 1, c, m, p, E);
        } else {
            double ep;
            uint32_t pp;
            orc_node_draw(kappa, slot, L - 1, c, ce - cs, &ep, &pp);
            orc_tree_expand(kappa, slot, V, L - 1, c, m + ep / (double)(ce - cs), cs + pp, E);
        }
    }
}

/* All V clocks of one slot. layout 0 = TREE, 1 = FLAT.  V must be in [1, 2^19]. */
int oracle_clocks(const uint32_t kappa[2], int slot, int V, int layout, double *E) {
    if (V < 1 || V > (1 << 19)) return -1;
    if (layout == 1) {
        for (int v = 0; v < V; v++) E[v] = orc_flat_clock(kappa, slot, v);
        return 0;
    }
    double ep;
    uint32_t p;
    orc_node_draw(kappa, slot, 5, 0u, (uint32_t)V, &ep, &p);
    orc_tree_expand(kappa, slot, (uint32_t)V, 5, 0u, ep / (double)V, p, E);
    return 0;
}

/* One clock by walking root -> token (TREE) or one word (FLAT). */
double oracle_clock(const uint32_t kappa[2], int slot, int V, int layout, int v) {
    if (layout == 1) return orc_flat_clock(kappa, slot, v);
    double ep;
    uint32_t p;
    orc_node_draw(kappa, slot, 5, 0u, (uint32_t)V, &ep, &p);
    double m = ep / (double)V;
    for (int L = 5; L >= 2; L--) {
        uint32_t c = (uint32_t)v >> ORC_SH[L - 1];
        uint32_t cs = orc_node_start(L - 1, c), ce = orc_node_end(L - 1, c, (uint32_t)V);
        if (!(p >= cs && p < ce)) {
            uint32_t pp;
            orc_node_draw(kappa, slot, L - 1, c, ce - cs, &ep, &pp);
            m = m + ep / (double)(ce - cs);
            p = cs + pp;
        }
    }
    if ((uint32_t)v == p) return m;
    return m + orc_token_draw(kappa, slot, (uint32_t)v);
}

/* ---------------- log-sum-exp and the race ------------------------------ */

/* L = ln sum_v exp(l_v / T), two passes in double; -inf for an empty row. */
double oracle_lse(const float *logits, int V, float T) {
    double M = -INFINITY;
    for (int v = 0; v < V; v++) {
        double x = (double)logits[v] / (double)T;
        if (x > M) M = x;
    }
    if (M == -INFINITY) return -INFINITY;
    double s = 0.0;
    for (int v = 0; v < V; v++) s += exp((double)logits[v] / (double)T - M);
    return M + log(s);
}

typedef struct {
    int32_t token;      /* winning token, -1 if no finite logit */
    int32_t slot;       /* winning slot (list index) */
    double best;        /* winning score  ln E - l/T */
    double second;      /* best score among all other tokens (+inf if none) */
    double lse;         /* ln sum exp(l/T) */
} oracle_race_result;

/* Race over slots [slot0, slot0 + nslots): score(v, j) = ln E_j[v] - l_v / T.
 * A draft row races its own slot (nslots = 1); the target row races all K slots
 * (augmented space V x [K]).  Exact ties: lowest v, then lowest j. */
int oracle_race(const float *logits, int V, float T, const uint32_t kappa[2], int slot0, int nslots,
                int layout, oracle_race_result *res) {
    if (V < 1 || V > (1 << 19) || nslots < 1) return -1;
    double *E = (double *)malloc(sizeof(double) * (size_t)V);
    double *tok_best = (double *)malloc(sizeof(double) * (size_t)V);
    int *tok_slot = (int *)malloc(sizeof(int) * (size_t)V);
    if (!E || !tok_best || !tok_slot) {
        free(E); free(tok_best); free(tok_slot);
        return -2;
    }
    for (int v = 0; v < V; v++) {
        tok_best[v] = INFINITY;
        tok_slot[v] = -1;
    }
    for (int j = slot0; j < slot0 + nslots; j++) {
        oracle_clocks(kappa, j, V, layout, E);
        for (int v = 0; v < V; v++) {
            double x = (double)logits[v] / (double)T;
            double s = (x == -INFINITY) ? INFINITY : log(E[v]) - x;
            if (s < tok_best[v]) {  /* strict: keeps the lowest slot on exact ties */
                tok_best[v] = s;
                tok_slot[v] = j;
            }
        }
    }
    int win = -1;
    double best = INFINITY;
    for (int v = 0; v < V; v++) {
        if (tok_best[v] < best) {  /* strict: keeps the lowest token on exact ties */
            best = tok_best[v];
            win = v;
        }
    }
    double second = INFINITY;
    for (int v = 0; v < V; v++)
        if (v != win && tok_best[v] < second) second = tok_best[v];
    res->token = win;
    res->slot = win >= 0 ? tok_slot[win] : -1;
    res->best = best;
    res->second = second;
    res->lse = oracle_lse(logits, V, T);
    free(E);
    free(tok_best);
    free(tok_slot);
    return 0;
}

/* ---------------- multi-sample PFR (identical drafters) ------------------ */

/* MPFR samples of one row (Sec. 5 eq. MPFR; App. "A better finite-support MPFR
 * implementation", Alg. "Direct finite-support implementation of B-sample MPFR"):
 * token v's arrivals are G_{v,j} = E_0[v] + ... + E_j[v] (slot i of the keyed
 * source is the (i+1)-th exponential of v's unit-rate clock), its mapped score is
 * G_{v,j} / P(v), and the samples are the labels of the smallest scores over
 * (v, j < nu) -- no token can hold more than nu of the nu smallest, so nu arrivals
 * per token suffice.  Scores in log form: ln G_{v,j} - l_v / T (the LSE is common
 * to all).  Exact ties: lowest v, then lowest j.
 * Writes the n_out smallest (score, token, arrival) in increasing order (n_out >= nu:
 * the first nu are the samples, the rest classify near-ties); entries past the
 * number of finite-score pairs get token -1 and score +inf.  Returns 0, or < 0 on
 * bad arguments / allocation failure. */
int oracle_mpfr(const float *logits, int V, float T, const uint32_t kappa[2], int nu, int layout, int n_out,
                int32_t *tokens, int32_t *arrivals, double *scores) {
    if (V < 1 || V > (1 << 19) || nu < 1 || n_out < nu) return -1;
    double *E = (double *)malloc(sizeof(double) * (size_t)V);
    double *G = (double *)malloc(sizeof(double) * (size_t)V * (size_t)nu);
    if (!E || !G) {
        free(E); free(G);
        return -2;
    }
    for (int j = 0; j < nu; j++) {
        oracle_clocks(kappa, j, V, layout, E);
        for (int v = 0; v < V; v++) G[(size_t)v * nu + j] = (j == 0 ? 0.0 : G[(size_t)v * nu + j - 1]) + E[v];
    }
    for (int i = 0; i < n_out; i++) {
        tokens[i] = -1;
        arrivals[i] = -1;
        scores[i] = INFINITY;
    }
    /* plain insertion into the sorted list of the n_out smallest */
    for (int v = 0; v < V; v++) {
        double x = (double)logits[v] / (double)T;
        if (x == -INFINITY) continue;
        for (int j = 0; j < nu; j++) {
            double sc = log(G[(size_t)v * nu + j]) - x;
            int pos = n_out;
            while (pos > 0) {
                int q = pos - 1;
                /* (sc, v, j) before entry q?  entries hold lower (v, j) on equal scores */
                if (sc < scores[q]) pos = q;
                else break;
            }
            if (pos >= n_out) continue;
            for (int q = n_out - 1; q > pos; q--) {
                scores[q] = scores[q - 1];
                tokens[q] = tokens[q - 1];
                arrivals[q] = arrivals[q - 1];
            }
            scores[pos] = sc;
            tokens[pos] = v;
            arrivals[pos] = j;
        }
    }
    free(E);
    free(G);
    return 0;
}

/* ---------------- detection --------------------------------------------- */

/* A_t = -log(1 - r_t(w_t)) with r = exp(-K * min_{j<K} E_j[w]): the target's
 * clock for token w in the augmented race is the minimum over the K slots
 * (Exp(K)), so r is uniform under H0.  For K = 1 this is Aaronson's score.
 * Returns NaN for a token outside [0, V) (not scored). */
double oracle_detect_term(uint64_t key, int m, int K, int V, int layout, const int32_t *tokens,
                          int64_t t) {
    int32_t win[64];
    if (m > 64) return NAN;
    for (int i = 0; i < m; i++) {
        int64_t idx = t - m + i;
        win[i] = idx >= 0 ? tokens[idx] : -1;
    }
    int32_t w = tokens[t];
    if (w < 0 || w >= V) return NAN;
    uint32_t kappa[2];
    oracle_context_key(key, t, win, m, kappa);
    double cmin = INFINITY;
    for (int j = 0; j < K; j++) {
        double e = oracle_clock(kappa, j, V, layout, w);
        if (e < cmin) cmin = e;
    }
    double c = (double)K * cmin;
    return -log(-expm1(-c));
}

/* The target's clock of the observed token, c_t = K * min_{j<K} E_j[w_t] (Exp(1)
 * under the null), whose pivot is r_t = exp(-c_t): every detection score below is
 * a function of it.  NaN for a token outside [0, V). */
double oracle_detect_clock(uint64_t key, int m, int K, int V, int layout, const int32_t *tokens, int64_t t) {
    int32_t win[64];
    if (m > 64) return NAN;
    for (int i = 0; i < m; i++) {
        int64_t idx = t - m + i;
        win[i] = idx >= 0 ? tokens[idx] : -1;
    }
    int32_t w = tokens[t];
    if (w < 0 || w >= V) return NAN;
    uint32_t kappa[2];
    oracle_context_key(key, t, win, m, kappa);
    double cmin = INFINITY;
    for (int j = 0; j < K; j++) {
        double e = oracle_clock(kappa, j, V, layout, w);
        if (e < cmin) cmin = e;
    }
    return (double)K * cmin;
}

/* Score one sequence: S = sum over t in [n0, n) of A_t (in t order), count of
 * scored tokens; per_token (nullable) receives every A_t (NaN when skipped). */
double oracle_detect_sequence(uint64_t key, int m, int K, int V, int layout, const int32_t *tokens,
                              int n, int n0, int32_t *count, double *per_token) {
    double S = 0.0;
    int32_t c = 0;
    for (int t = 0; t < n; t++) {
        if (t < n0) {
            if (per_token) per_token[t] = NAN;
            continue;
        }
        double a = oracle_detect_term(key, m, K, V, layout, tokens, t);
        if (per_token) per_token[t] = a;
        if (a == a) {
            S += a;
            c++;
        }
    }
    *count = c;
    return S;
}
