/*
 * HiLS attention -- CPU reference oracle.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke check and the
 * CPU-baseline leg of the benchmark load this library; the GPU library never
 * links, includes or calls it, and it shares no code with the GPU kernels.
 *
 * This is a plain, slow, step-by-step statement of what HiLS attention
 * computes, written from the paper (arXiv 2607.02980):
 *
 *   Sec. 2.1      chunk partition c(j) = floor(j / S); the chunk-aligned left
 *                 edge of the local window l(i) = floor((i - W + 1) / S) * S;
 *                 the candidate chunks C_i = {0, ..., l(i)/S - 1}.
 *   Eq. (1)       local-window mass Z_swa = sum_{j = l(i)}^{i} exp(s_ij).
 *   Eq. (9)       surrogate score s^_ic = q_i . k'_c / sqrt(d) + b'_c, the
 *                 top-K selection I_i, the surrogate mass.
 *   Eq. (10)      hierarchical softmax: intra-chunk softmax times the
 *                 inter-chunk surrogate share; the local window takes Z_swa
 *                 as its own mass.
 *   Eq. (11)      Q-Cal: a routing query q^ (here the optional `q_route`)
 *                 is used only inside the surrogate score.
 *   Prop. 3.1    landmark compression: k'_c = attention of the landmark query
 *                 q'_c over its chunk's keys, b'_c = the entropy of that
 *                 attention (and its backward).
 *   Sec. 4.1 ("HiLS-Attention in GQA") and Appendix C: one selection per
 *                 KV group, ranked by the maximum of the per-head surrogate
 *                 scores; fusion weights stay per head.
 *
 * The backward is the derivative of Eq. (10) with the selection held fixed
 * (the top-K set is piecewise constant; Sec. 9 notes that unselected chunks
 * receive no gradient).
 *
 * Readings where the paper is silent or garbled (all listed in the design
 * notes of the repository):
 *   - l(i) < 0 (i < W - 1) is clamped to 0: C_i is empty, attention is local.
 *   - Appendix C writes "argmax_h"; the text says "taking the maximum", so the
 *     group score is the max VALUE over the group's heads.
 *   - Appendix C sums Z^h_swa over T_c; Eq. (1) and the weight cases of
 *     Appendix C put the window at [l(i), i], which is used here.
 *   - rank-descending ties are broken toward the smaller chunk index.
 *   - |C_i| < K selects all of C_i; idx is padded with -1.
 *   - one `scale` multiplies both the token logits and the surrogate score.
 *   - landmark heads: Hl == Hq (one compressed key per query head, App. C)
 *     or Hl == Hkv (one per KV group); the bias b'_c has the same heads.
 *
 * Precision: the file is compiled twice, REAL=double (the reference used for
 * every pin and every parity check) and REAL=float (the plain fp32 oracle).
 * Inputs are float arrays (bf16 data is widened exactly); outputs are REAL.
 *
 * Layouts (row-major, contiguous):
 *   q, q_route, out, dq, dq_route : [B, Hq,  N, d]
 *   k, v, dk, dv                  : [B, Hkv, L, d]
 *   lmk, dlmk                     : [B, Hl,  L/S, d]
 *   bias, dbias                   : [B, Hl,  L/S]
 *   lse                           : [B, Hq,  N]
 *   idx                           : [B, Hkv, N, K]   ascending, -1 padded
 *   sel_score                     : [B, Hq,  N, K]   s^ of idx entries
 *   alpha                         : [B, Hq,  N, K+1] fusion weights, slot 0 = local
 *   qpos                          : [B, N]  position of each query in its
 *                                   sequence (NULL: query n sits at n)
 *   rows                          : nrows pairs (b, n) to process (NULL: all)
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifndef REAL
#define REAL double
#endif
#ifndef SUFFIX
#define SUFFIX f64
#endif
#define CAT2(a, b) a##_##b
#define CAT(a, b) CAT2(a, b)
#define API(name) CAT(hils_oracle_##name, SUFFIX)

#if REAL_IS_FLOAT
#define EXP expf
#define LOG logf
#else
#define EXP exp
#define LOG log
#endif

typedef struct {
    int B, Hq, Hkv, Hl;
    int N;      /* queries per sequence */
    int L;      /* key positions per sequence (the landmark rows are L / S) */
    int d;
    int chunk;  /* S */
    int topk;   /* K */
    int window; /* W */
    double scale;
    int head_norm; /* 1: rank by per-head normalised scores (Sec. 4.1 variant) */
} hils_oracle_shape;

/* ---- small helpers --------------------------------------------------- */

static long floor_div(long a, long b) {
    long q = a / b;
    if ((a % b != 0) && ((a < 0) != (b < 0))) q -= 1;
    return q;
}

/* Number of candidate chunks |C_i| = l(i) / S for a query at position i. */
static long n_candidates(long i, long S, long W) {
    long lc = floor_div(i - W + 1, S);
    return lc < 0 ? 0 : lc;
}

static REAL dot_f(const float* a, const float* b, int d) {
    REAL s = 0;
    for (int t = 0; t < d; ++t) s += (REAL)a[t] * (REAL)b[t];
    return s;
}

static REAL logsumexp(const REAL* x, long n) {
    REAL m = -INFINITY;
    for (long t = 0; t < n; ++t)
        if (x[t] > m) m = x[t];
    REAL s = 0;
    for (long t = 0; t < n; ++t) s += EXP(x[t] - m);
    return m + LOG(s);
}

typedef struct {
    const hils_oracle_shape* p;
    const float *q, *k, *v, *lmk, *bias, *q_route;
    const int32_t* qpos;
} inputs;

static long nchunks_of(const hils_oracle_shape* p) { return p->L / p->chunk; }

static const float* Q(const inputs* in, int b, int h, int n) {
    const hils_oracle_shape* p = in->p;
    return in->q + (((size_t)b * p->Hq + h) * p->N + n) * p->d;
}
static const float* QHAT(const inputs* in, int b, int h, int n) {
    const hils_oracle_shape* p = in->p;
    const float* base = in->q_route ? in->q_route : in->q;
    return base + (((size_t)b * p->Hq + h) * p->N + n) * p->d;
}
static const float* KEY(const inputs* in, int b, int g, long j) {
    const hils_oracle_shape* p = in->p;
    return in->k + (((size_t)b * p->Hkv + g) * p->L + j) * p->d;
}
static const float* VAL(const inputs* in, int b, int g, long j) {
    const hils_oracle_shape* p = in->p;
    return in->v + (((size_t)b * p->Hkv + g) * p->L + j) * p->d;
}
/* landmark head that serves query head h: h itself (Hl == Hq) or its group. */
static int lmk_head(const hils_oracle_shape* p, int h) {
    return p->Hl == p->Hq ? h : h / (p->Hq / p->Hkv);
}
static const float* LMK(const inputs* in, int b, int hl, long c) {
    const hils_oracle_shape* p = in->p;
    return in->lmk + (((size_t)b * p->Hl + hl) * nchunks_of(p) + c) * p->d;
}
static REAL BIAS(const inputs* in, int b, int hl, long c) {
    const hils_oracle_shape* p = in->p;
    if (!in->bias) return 0;
    return (REAL)in->bias[((size_t)b * p->Hl + hl) * nchunks_of(p) + c];
}
static long position_of(const inputs* in, int b, int n) {
    return in->qpos ? (long)in->qpos[(size_t)b * in->p->N + n] : (long)n;
}

/* Eq. (9) with Eq. (11): per-head surrogate score of chunk c for query head h. */
static REAL surrogate_score(const inputs* in, int b, int h, int n, long c) {
    const hils_oracle_shape* p = in->p;
    int hl = lmk_head(p, h);
    return (REAL)p->scale * dot_f(QHAT(in, b, h, n), LMK(in, b, hl, c), p->d) + BIAS(in, b, hl, c);
}

/* Appendix C: group score = max over the G heads of group g.
 * head_norm (the wording of Sec. 4.1, "normalized chunk weights" per head before
 * the maximum): each head's scores are first turned into log-weights over the
 * candidates, s^_hc - log sum_{c' in C_i} exp(s^_hc'), so that a head whose
 * scores are all large does not outrank a head with one decisive chunk. */
static void group_scores(const inputs* in, int b, int g, int n, long ncand, REAL* sigma) {
    const hils_oracle_shape* p = in->p;
    int G = p->Hq / p->Hkv;
    REAL* sh = (REAL*)malloc(sizeof(REAL) * (ncand > 0 ? ncand : 1));
    for (long c = 0; c < ncand; ++c) sigma[c] = -INFINITY;
    for (int hh = 0; hh < G; ++hh) {
        for (long c = 0; c < ncand; ++c) sh[c] = surrogate_score(in, b, g * G + hh, n, c);
        const REAL lse = p->head_norm && ncand > 0 ? logsumexp(sh, ncand) : 0;
        for (long c = 0; c < ncand; ++c)
            if (sh[c] - lse > sigma[c]) sigma[c] = sh[c] - lse;
    }
    free(sh);
}

/* Eq. (9): I_i = {c in C_i : rank_desc(sigma_c) < K}.  Ties go to the smaller
 * index.  Done the obvious way: K passes of "take the best remaining".
 * Returns the count and writes the chosen chunks in ascending order. */
static int select_topk(const REAL* sigma, long ncand, int K, int32_t* chosen) {
    char* taken = (char*)calloc(ncand > 0 ? ncand : 1, 1);
    int cnt = 0;
    for (int r = 0; r < K && r < ncand; ++r) {
        long best = -1;
        for (long c = 0; c < ncand; ++c) {
            if (taken[c]) continue;
            if (best < 0 || sigma[c] > sigma[best]) best = c; /* strict: keeps smaller c on ties */
        }
        taken[best] = 1;
        cnt++;
    }
    int w = 0;
    for (long c = 0; c < ncand; ++c)
        if (taken[c]) chosen[w++] = (int32_t)c;
    free(taken);
    return cnt;
}

/* Scaled token logits s_ij = scale * q_i . k_j for j in [j0, j1). */
static void token_logits(const inputs* in, const float* qv, int b, int g, long j0, long j1, REAL* s) {
    for (long j = j0; j < j1; ++j) s[j - j0] = (REAL)in->p->scale * dot_f(qv, KEY(in, b, g, j), in->p->d);
}

/* Softmax attention over keys [j0, j1): returns the LSE of the logits and the
 * normalised output o = sum_j softmax(s)_j v_j. */
static REAL softmax_attend(const inputs* in, const float* qv, int b, int g, long j0, long j1, REAL* o, REAL* work) {
    const int d = in->p->d;
    long n = j1 - j0;
    token_logits(in, qv, b, g, j0, j1, work);
    REAL lse = logsumexp(work, n);
    for (int t = 0; t < d; ++t) o[t] = 0;
    for (long j = j0; j < j1; ++j) {
        REAL pj = EXP(work[j - j0] - lse);
        const float* vj = VAL(in, b, g, j);
        for (int t = 0; t < d; ++t) o[t] += pj * (REAL)vj[t];
    }
    return lse;
}

/* Everything the forward knows about one (b, n, head h) once the selection I is fixed. */
typedef struct {
    long pos, ell;         /* query position i and window edge l(i) */
    int nsel;              /* |I_i| */
    int32_t sel[1024];     /* I_i ascending (K <= 1024) */
    REAL shat[1024];       /* s^_h of each selected chunk */
    REAL lam0;             /* log Z_swa (Eq. (1)) */
    REAL lse_c[1024];      /* log Z_c of each selected chunk */
    REAL L;                /* log of the surrogate partition function */
    REAL alpha0, alpha[1024];
} row_state;

/* ---- forward ---------------------------------------------------------- */

static int forward_row(const inputs* in, int b, int n, int given_idx, int32_t* idx, REAL* out, REAL* lse,
                       REAL* sel_score, REAL* alpha_out) {
    const hils_oracle_shape* p = in->p;
    const int G = p->Hq / p->Hkv, S = p->chunk, K = p->topk, W = p->window, d = p->d;
    const long i = position_of(in, b, n);
    const long ncand = n_candidates(i, S, W);
    const long ell = ncand * S; /* Sec. 2.1, clamped at 0 */
    REAL* sigma = (REAL*)malloc(sizeof(REAL) * (ncand > 0 ? ncand : 1));
    REAL* work = (REAL*)malloc(sizeof(REAL) * (size_t)(i - ell + 1 + S));
    REAL* o0 = (REAL*)malloc(sizeof(REAL) * d);
    REAL* oc = (REAL*)malloc(sizeof(REAL) * (size_t)d * (K > 0 ? K : 1));
    row_state* st = (row_state*)malloc(sizeof(row_state));
    int rc = 0;

    for (int g = 0; g < p->Hkv && rc == 0; ++g) {
        int32_t* idx_row = idx + (((size_t)b * p->Hkv + g) * p->N + n) * K;
        /* steps 1-4: candidate scores, group max, top-K */
        if (given_idx) {
            st->nsel = 0;
            for (int r = 0; r < K; ++r) {
                int32_t c = idx_row[r];
                if (c < 0) continue;
                if (c >= ncand) { rc = -2; break; }         /* not a candidate of this query */
                if (st->nsel > 0 && c <= st->sel[st->nsel - 1]) { rc = -3; break; } /* must ascend */
                st->sel[st->nsel++] = c;
            }
        } else {
            group_scores(in, b, g, n, ncand, sigma);
            st->nsel = select_topk(sigma, ncand, K, st->sel);
            for (int r = 0; r < K; ++r) idx_row[r] = r < st->nsel ? st->sel[r] : -1;
        }
        if (rc) break;

        for (int hh = 0; hh < G; ++hh) {
            const int h = g * G + hh;
            const float* qv = Q(in, b, h, n);
            /* step 5: local window [l(i), i] -- Eq. (1) */
            REAL lam0 = softmax_attend(in, qv, b, g, ell, i + 1, o0, work);
            /* step 6: intra-chunk softmax inside every selected chunk -- Eq. (10) */
            for (int r = 0; r < st->nsel; ++r) {
                long c = st->sel[r];
                st->lse_c[r] = softmax_attend(in, qv, b, g, c * S, c * S + S, oc + (size_t)r * d, work);
                st->shat[r] = surrogate_score(in, b, h, n, c);
            }
            /* step 7: inter-chunk softmax over {s^_c : c in I} U {log Z_swa} -- Eqs. (9), (10) */
            REAL logits[1025];
            logits[0] = lam0;
            for (int r = 0; r < st->nsel; ++r) logits[1 + r] = st->shat[r];
            REAL Lz = logsumexp(logits, st->nsel + 1);
            REAL* orow = out + (((size_t)b * p->Hq + h) * p->N + n) * d;
            REAL a0 = EXP(lam0 - Lz);
            for (int t = 0; t < d; ++t) orow[t] = a0 * o0[t];
            for (int r = 0; r < st->nsel; ++r) {
                REAL ar = EXP(st->shat[r] - Lz);
                for (int t = 0; t < d; ++t) orow[t] += ar * oc[(size_t)r * d + t];
            }
            lse[((size_t)b * p->Hq + h) * p->N + n] = Lz;
            if (sel_score) {
                REAL* srow = sel_score + (((size_t)b * p->Hq + h) * p->N + n) * K;
                for (int r = 0; r < K; ++r) srow[r] = r < st->nsel ? st->shat[r] : (REAL)-INFINITY;
            }
            if (alpha_out) {
                REAL* arow = alpha_out + (((size_t)b * p->Hq + h) * p->N + n) * (K + 1);
                arow[0] = a0;
                for (int r = 0; r < K; ++r) arow[1 + r] = r < st->nsel ? EXP(st->shat[r] - Lz) : 0;
            }
        }
    }
    free(sigma); free(work); free(o0); free(oc); free(st);
    return rc;
}

static int check_shape(const hils_oracle_shape* p) {
    if (p->B < 1 || p->Hq < 1 || p->Hkv < 1 || p->N < 1 || p->L < 1 || p->d < 1) return -1;
    if (p->Hq % p->Hkv) return -1;
    if (p->Hl != p->Hq && p->Hl != p->Hkv) return -1;
    if (p->chunk < 1 || p->topk < 1 || p->topk > 1024 || p->window < 1) return -1;
    if (p->L % p->chunk) return -1;
    return 0;
}

static int check_positions(const inputs* in) {
    const hils_oracle_shape* p = in->p;
    for (int b = 0; b < p->B; ++b)
        for (int n = 0; n < p->N; ++n) {
            long i = position_of(in, b, n);
            if (i < 0 || i >= p->L) return -4;
        }
    return 0;
}

/* Forward.  Writes out/lse (and idx unless given_idx) for the listed rows.
 * Returns 0, or a negative code: -1 bad shape, -2 a given index is not a
 * candidate of its query, -3 given indices not strictly ascending, -4 a query
 * position outside [0, L). */
int API(fwd)(const hils_oracle_shape* p, const float* q, const float* k, const float* v, const float* lmk,
             const float* bias, const float* q_route, const int32_t* qpos, const int32_t* rows, int nrows,
             int given_idx, int32_t* idx, REAL* out, REAL* lse, REAL* sel_score, REAL* alpha) {
    if (check_shape(p)) return -1;
    inputs in = {p, q, k, v, lmk, bias, q_route, qpos};
    int rc = check_positions(&in);
    if (rc) return rc;
    long total = rows ? nrows : (long)p->B * p->N;
    int err = 0;
#pragma omp parallel for schedule(dynamic, 4) reduction(min : err)
    for (long r = 0; r < total; ++r) {
        int b = rows ? rows[2 * r] : (int)(r / p->N);
        int n = rows ? rows[2 * r + 1] : (int)(r % p->N);
        int e = forward_row(&in, b, n, given_idx, idx, out, lse, sel_score, alpha);
        if (e < err) err = e;
    }
    return err;
}

/* Group scores sigma_c (Appendix C) of one query for c in C_i; returns |C_i|
 * (sigma must hold L/S entries). */
long API(group_scores)(const hils_oracle_shape* p, const float* q, const float* lmk, const float* bias,
                       const float* q_route, const int32_t* qpos, int b, int g, int n, REAL* sigma) {
    if (check_shape(p)) return -1;
    inputs in = {p, q, NULL, NULL, lmk, bias, q_route, qpos};
    long i = position_of(&in, b, n);
    long ncand = n_candidates(i, p->chunk, p->window);
    group_scores(&in, b, g, n, ncand, sigma);
    return ncand;
}

/* Dense weight form (Appendix C, the case-wise definition of w^h_ij): writes
 * w [B, Hq, N, L] for a given selection idx.  Used to check the factored
 * forward against the paper's second formulation on tiny shapes. */
int API(dense_weights)(const hils_oracle_shape* p, const float* q, const float* k, const float* lmk,
                       const float* bias, const float* q_route, const int32_t* qpos, const int32_t* idx,
                       REAL* w) {
    if (check_shape(p)) return -1;
    inputs in = {p, q, k, NULL, lmk, bias, q_route, qpos};
    const int G = p->Hq / p->Hkv, S = p->chunk, K = p->topk;
    REAL* s = (REAL*)malloc(sizeof(REAL) * p->L);
    for (int b = 0; b < p->B; ++b)
        for (int n = 0; n < p->N; ++n) {
            long i = position_of(&in, b, n);
            long ell = n_candidates(i, S, p->window) * S;
            for (int h = 0; h < p->Hq; ++h) {
                int g = h / G;
                const int32_t* sel = idx + (((size_t)b * p->Hkv + g) * p->N + n) * K;
                REAL* wrow = w + (((size_t)b * p->Hq + h) * p->N + n) * p->L;
                for (long j = 0; j < p->L; ++j) wrow[j] = 0;
                token_logits(&in, Q(&in, b, h, n), b, g, 0, i + 1, s);
                /* Z^h_swa over [l(i), i];  Z^h_c over the S keys of chunk c */
                REAL Zswa = 0;
                for (long j = ell; j <= i; ++j) Zswa += EXP(s[j]);
                REAL Zhat = Zswa;
                for (int r = 0; r < K; ++r)
                    if (sel[r] >= 0) Zhat += EXP(surrogate_score(&in, b, h, n, sel[r]));
                for (long j = ell; j <= i; ++j) wrow[j] = EXP(s[j]) / Zhat;
                for (int r = 0; r < K; ++r) {
                    long c = sel[r];
                    if (c < 0) continue;
                    REAL Zc = 0;
                    for (long j = c * S; j < c * S + S; ++j) Zc += EXP(s[j]);
                    REAL share = EXP(surrogate_score(&in, b, h, n, c)) / Zhat;
                    for (long j = c * S; j < c * S + S; ++j) wrow[j] = EXP(s[j]) / Zc * share;
                }
            }
        }
    free(s);
    return 0;
}

/* ---- backward --------------------------------------------------------- */

/* Gradient contributions of one row (b, n) for KV group g, selection fixed to idx.
 * With g = dO, u = g . out:
 *   local key j:      w_j = exp(s_j - L);            dv_j += w_j g;  ds_j = w_j (g.v_j - u)
 *   chunk c, key j:   p_j = exp(s_j - log Z_c), a_c = exp(s^_c - L), u_c = g . o_c;
 *                     dv_j += a_c p_j g;  ds_j = a_c p_j (g.v_j - u_c)
 *   retrieval score:  ds^_c = a_c (u_c - u)
 *   dq += scale ds_j k_j;  dk_j += scale ds_j q;
 *   dq^ += scale ds^_c k'_c;  dk'_c += scale ds^_c q^;  db'_c += ds^_c. */
static void backward_row(const inputs* in, int b, int g, int n, const int32_t* idx, const float* dout, REAL* dq,
                         REAL* dk, REAL* dv, REAL* dlmk, REAL* dbias, REAL* dq_route) {
    const hils_oracle_shape* p = in->p;
    const int G = p->Hq / p->Hkv, S = p->chunk, K = p->topk, d = p->d;
    const long i = position_of(in, b, n);
    const long ell = n_candidates(i, S, p->window) * S;
    const long nloc = i - ell + 1;
    const long nch = nchunks_of(p);
    const int32_t* idx_row = idx + (((size_t)b * p->Hkv + g) * p->N + n) * K;
    int nsel = 0;
    int32_t sel[1024];
    for (int r = 0; r < K; ++r)
        if (idx_row[r] >= 0) sel[nsel++] = idx_row[r];

    REAL* sl = (REAL*)malloc(sizeof(REAL) * nloc);
    REAL* sc = (REAL*)malloc(sizeof(REAL) * (size_t)(nsel > 0 ? nsel : 1) * S);
    REAL* lse_c = (REAL*)malloc(sizeof(REAL) * (nsel + 1));
    REAL* shat = (REAL*)malloc(sizeof(REAL) * (nsel + 1));
    REAL* oc = (REAL*)malloc(sizeof(REAL) * (size_t)(nsel + 1) * d);
    REAL* out = (REAL*)malloc(sizeof(REAL) * d);
    REAL* gq = (REAL*)malloc(sizeof(REAL) * d);
    REAL* gqhat = (REAL*)malloc(sizeof(REAL) * d);

    for (int hh = 0; hh < G; ++hh) {
        const int h = g * G + hh;
        const int hl = lmk_head(p, h);
        const float* qv = Q(in, b, h, n);
        const float* qh = QHAT(in, b, h, n);
        const float* gd = dout + (((size_t)b * p->Hq + h) * p->N + n) * d;
        /* recompute the forward of this row */
        token_logits(in, qv, b, g, ell, i + 1, sl);
        REAL lam0 = logsumexp(sl, nloc);
        for (int r = 0; r < nsel; ++r) {
            long c = sel[r];
            token_logits(in, qv, b, g, c * S, c * S + S, sc + (size_t)r * S);
            lse_c[r] = logsumexp(sc + (size_t)r * S, S);
            shat[r] = surrogate_score(in, b, h, n, c);
        }
        REAL logits[1025];
        logits[0] = lam0;
        for (int r = 0; r < nsel; ++r) logits[1 + r] = shat[r];
        REAL Lz = logsumexp(logits, nsel + 1);
        for (int t = 0; t < d; ++t) out[t] = 0;
        for (long j = ell; j <= i; ++j) {
            REAL w = EXP(sl[j - ell] - Lz);
            const float* vj = VAL(in, b, g, j);
            for (int t = 0; t < d; ++t) out[t] += w * vj[t];
        }
        for (int r = 0; r < nsel; ++r) {
            REAL a = EXP(shat[r] - Lz);
            long c = sel[r];
            for (int t = 0; t < d; ++t) oc[(size_t)r * d + t] = 0;
            for (long j = c * S; j < c * S + S; ++j) {
                REAL pj = EXP(sc[(size_t)r * S + (j - c * S)] - lse_c[r]);
                const float* vj = VAL(in, b, g, j);
                for (int t = 0; t < d; ++t) oc[(size_t)r * d + t] += pj * vj[t];
            }
            for (int t = 0; t < d; ++t) out[t] += a * oc[(size_t)r * d + t];
        }
        REAL ubar = 0;
        for (int t = 0; t < d; ++t) ubar += (REAL)gd[t] * out[t];
        for (int t = 0; t < d; ++t) gq[t] = gqhat[t] = 0;

        /* local window */
        for (long j = ell; j <= i; ++j) {
            REAL w = EXP(sl[j - ell] - Lz);
            const float* vj = VAL(in, b, g, j);
            const float* kj = KEY(in, b, g, j);
            REAL gv = dot_f(gd, vj, d);
            REAL ds = w * (gv - ubar);
            REAL* dvj = dv + (((size_t)b * p->Hkv + g) * p->L + j) * d;
            REAL* dkj = dk + (((size_t)b * p->Hkv + g) * p->L + j) * d;
            for (int t = 0; t < d; ++t) {
                dvj[t] += w * gd[t];
                dkj[t] += p->scale * ds * qv[t];
                gq[t] += p->scale * ds * kj[t];
            }
        }
        /* selected chunks */
        for (int r = 0; r < nsel; ++r) {
            long c = sel[r];
            REAL a = EXP(shat[r] - Lz);
            REAL uc = 0;
            for (int t = 0; t < d; ++t) uc += (REAL)gd[t] * oc[(size_t)r * d + t];
            for (long j = c * S; j < c * S + S; ++j) {
                REAL pj = EXP(sc[(size_t)r * S + (j - c * S)] - lse_c[r]);
                const float* vj = VAL(in, b, g, j);
                const float* kj = KEY(in, b, g, j);
                REAL gv = dot_f(gd, vj, d);
                REAL ds = a * pj * (gv - uc);
                REAL* dvj = dv + (((size_t)b * p->Hkv + g) * p->L + j) * d;
                REAL* dkj = dk + (((size_t)b * p->Hkv + g) * p->L + j) * d;
                for (int t = 0; t < d; ++t) {
                    dvj[t] += a * pj * gd[t];
                    dkj[t] += p->scale * ds * qv[t];
                    gq[t] += p->scale * ds * kj[t];
                }
            }
            REAL dshat = a * (uc - ubar);
            const float* lc = LMK(in, b, hl, c);
            REAL* dlc = dlmk + (((size_t)b * p->Hl + hl) * nch + c) * d;
            for (int t = 0; t < d; ++t) {
                gqhat[t] += p->scale * dshat * lc[t];
                dlc[t] += p->scale * dshat * qh[t];
            }
            if (dbias) dbias[((size_t)b * p->Hl + hl) * nch + c] += dshat;
        }
        REAL* dqrow = dq + (((size_t)b * p->Hq + h) * p->N + n) * d;
        REAL* dqhrow = dq_route ? dq_route + (((size_t)b * p->Hq + h) * p->N + n) * d : dqrow;
        for (int t = 0; t < d; ++t) {
            dqrow[t] += gq[t];
            dqhrow[t] += gqhat[t];
        }
    }
    free(sl); free(sc); free(lse_c); free(shat); free(oc); free(out); free(gq); free(gqhat);
}

/* Backward.  Accumulates (+=) into dq, dk, dv, dlmk, dbias (may be NULL) and
 * dq_route (NULL: the routing-query gradient is added to dq) the
 * contributions of the listed rows (NULL: all rows), with idx as selected by
 * the forward.  only_group >= 0 restricts the work to that KV group (a
 * sampled check of one group's gradients).  Returns 0 or a negative code as
 * for the forward. */
int API(bwd)(const hils_oracle_shape* p, const float* dout, const float* q, const float* k, const float* v,
             const float* lmk, const float* bias, const float* q_route, const int32_t* qpos, const int32_t* rows,
             int nrows, const int32_t* idx, REAL* dq, REAL* dk, REAL* dv, REAL* dlmk, REAL* dbias,
             REAL* dq_route, int only_group) {
    if (check_shape(p)) return -1;
    inputs in = {p, q, k, v, lmk, bias, q_route, qpos};
    int rc = check_positions(&in);
    if (rc) return rc;
    long total = rows ? nrows : (long)p->B * p->N;
    /* Parallel over (b, g): every write of a row of group g lands in
     * group g's slices (dk, dv, and dlmk/dbias heads of g), so there are no races. */
#pragma omp parallel for schedule(dynamic, 1)
    for (long bg = 0; bg < (long)p->B * p->Hkv; ++bg) {
        int b = (int)(bg / p->Hkv), g = (int)(bg % p->Hkv);
        if (only_group >= 0 && g != only_group) continue;
        for (long r = 0; r < total; ++r) {
            int rb = rows ? rows[2 * r] : (int)(r / p->N);
            int rn = rows ? rows[2 * r + 1] : (int)(r % p->N);
            if (rb != b) continue;
            backward_row(&in, b, g, rn, idx, dout, dq, dk, dv, dlmk, dbias, dq_route);
        }
    }
    return 0;
}

/* ---- landmark compression (Prop. 3.1; the section's NEXT step) --------------
 *
 * For landmark head hl (KV group g(hl): hl / (Hl / Hkv)) and chunk c with keys
 * k_j, j in [cS, cS + S), and its landmark query q'_c:
 *   s_j = scale * q'_c . k_j,   p = softmax(s),
 *   k'_c = sum_j p_j k_j        (an attention of q'_c over the chunk's own keys),
 *   b'_c = - sum_j p_j log p_j  (the entropy of p),
 * with log p_j taken as s_j - LSE(s), which equals it exactly and stays finite
 * when p_j underflows.
 *
 * Layouts: lq, lmk, dlq, dlmk : [B, Hl, L/S, d];  bias, dbias : [B, Hl, L/S];
 * k, dk : [B, Hkv, L, d]. */

static int lmk_group(const hils_oracle_shape* p, int hl) { return hl / (p->Hl / p->Hkv); }

/* Forward: writes lmk and bias for every (b, hl, c).  Returns 0 or -1 (shape). */
int API(landmark_fwd)(const hils_oracle_shape* p, const float* lq, const float* k, REAL* lmk, REAL* bias) {
    if (check_shape(p)) return -1;
    const long nc = nchunks_of(p), S = p->chunk;
    const int d = p->d;
#pragma omp parallel for schedule(dynamic, 4)
    for (long t = 0; t < (long)p->B * p->Hl * nc; ++t) {
        const int b = (int)(t / ((long)p->Hl * nc)), hl = (int)(t / nc % p->Hl);
        const long c = t % nc;
        const int g = lmk_group(p, hl);
        const float* qc = lq + (((size_t)b * p->Hl + hl) * nc + c) * d;
        REAL* s = (REAL*)malloc(sizeof(REAL) * S);
        for (long j = 0; j < S; ++j)
            s[j] = p->scale * dot_f(qc, k + (((size_t)b * p->Hkv + g) * p->L + c * S + j) * d, d);
        const REAL lse = logsumexp(s, S);
        REAL* kc = lmk + (((size_t)b * p->Hl + hl) * nc + c) * d;
        for (int u = 0; u < d; ++u) kc[u] = 0;
        REAL ent = 0;
        for (long j = 0; j < S; ++j) {
            const REAL logp = s[j] - lse, pj = EXP(logp);
            const float* kj = k + (((size_t)b * p->Hkv + g) * p->L + c * S + j) * d;
            for (int u = 0; u < d; ++u) kc[u] += pj * (REAL)kj[u];
            ent -= pj * logp;
        }
        bias[((size_t)b * p->Hl + hl) * nc + c] = ent;
        free(s);
    }
    return 0;
}

/* Backward of the compression for upstream gradients dlmk (of k'_c) and dbias
 * (of b'_c, NULL = 0).  By the chain rule through the two outputs:
 *   dL/dp_j = dk'_c . k_j - db'_c (log p_j + 1),
 *   dL/ds_j = p_j (dL/dp_j - sum_m p_m dL/dp_m)            (softmax Jacobian),
 *   dq'_c   = scale * sum_j dL/ds_j k_j,
 *   dk_j   += p_j dk'_c + scale * dL/ds_j q'_c              (k_j appears in k'_c and in s_j).
 * Writes dlq; accumulates (+=) into dk over the landmark heads of each group.
 * Returns 0 or -1. */
int API(landmark_bwd)(const hils_oracle_shape* p, const float* lq, const float* k, const float* dlmk,
                      const float* dbias, REAL* dlq, REAL* dk) {
    if (check_shape(p)) return -1;
    const long nc = nchunks_of(p), S = p->chunk;
    const int d = p->d, per_group = p->Hl / p->Hkv;
    /* parallel over (b, g, c): the landmark heads of a group write the same dk rows */
#pragma omp parallel for schedule(dynamic, 4)
    for (long t = 0; t < (long)p->B * p->Hkv * nc; ++t) {
        const int b = (int)(t / ((long)p->Hkv * nc)), g = (int)(t / nc % p->Hkv);
        const long c = t % nc;
        REAL* s = (REAL*)malloc(sizeof(REAL) * S);
        REAL* pr = (REAL*)malloc(sizeof(REAL) * S);
        REAL* gp = (REAL*)malloc(sizeof(REAL) * S);
        for (int hl = g * per_group; hl < (g + 1) * per_group; ++hl) {
            const size_t row = ((size_t)b * p->Hl + hl) * nc + c;
            const float* qc = lq + row * d;
            const float* dkc = dlmk + row * d;
            const REAL db = dbias ? (REAL)dbias[row] : 0;
            for (long j = 0; j < S; ++j)
                s[j] = p->scale * dot_f(qc, k + (((size_t)b * p->Hkv + g) * p->L + c * S + j) * d, d);
            const REAL lse = logsumexp(s, S);
            REAL mean = 0;
            for (long j = 0; j < S; ++j) {
                const float* kj = k + (((size_t)b * p->Hkv + g) * p->L + c * S + j) * d;
                const REAL logp = s[j] - lse;
                pr[j] = EXP(logp);
                gp[j] = dot_f(dkc, kj, d) - db * (logp + 1);
                mean += pr[j] * gp[j];
            }
            REAL* dq = dlq + row * d;
            for (int u = 0; u < d; ++u) dq[u] = 0;
            for (long j = 0; j < S; ++j) {
                const float* kj = k + (((size_t)b * p->Hkv + g) * p->L + c * S + j) * d;
                REAL* dkj = dk + (((size_t)b * p->Hkv + g) * p->L + c * S + j) * d;
                const REAL ds = pr[j] * (gp[j] - mean);
                for (int u = 0; u < d; ++u) {
                    dq[u] += p->scale * ds * (REAL)kj[u];
                    dkj[u] += pr[j] * (REAL)dkc[u] + p->scale * ds * (REAL)qc[u];
                }
            }
        }
        free(s); free(pr); free(gp);
    }
    return 0;
}
