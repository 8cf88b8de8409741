/*
 * Serial CPU oracle for WFST Viterbi beam decoding with state-level lattices.
 *
 * TEST INFRASTRUCTURE ONLY: the decoder never calls this code and shares
 * nothing with it.  See oracle_wfst.h for the interface.
 *
 * The method, as read from Z. Chen, "Linguistic Search Optimization for Deep
 * Learning Based LVCSR":
 *
 *  - Costs are negative log probabilities, so the arg max of Eq. 1 becomes a
 *    minimum-cost path (tropical semiring).  A candidate cost through an
 *    emitting arc is (previous cost + arc weight) - log-likelihood of the
 *    arc's input label at the current frame, two float32 roundings in that
 *    order.
 *  - Token passing (Sec. 3): every active state holds one token (cost,
 *    predecessor arc).  Each frame, every token is passed along its
 *    emitting out-arcs and every state keeps the minimum over its incoming
 *    candidates ("token recombination", Sec. 3).  Ties on the cost are
 *    broken towards the lower arc index; the start token (no arc) wins all
 *    ties.  Epsilon arcs consume no frame and are closed after each frame.
 *  - Viterbi beam search (Sec. 1, Alg. 1): after each frame only tokens
 *    within `beam` of the best survive; with a max-active limit only the
 *    max_active best (ties at the limit kept) survive.
 *  - Label-synchronous decoding (Sec. 2, Alg. 1): a frame is blank when the
 *    blank posterior exceeds the threshold (the set U); blank frames leave
 *    the token set untouched (Eq. 2 drops their factors), so the search runs
 *    on the T - |U| remaining frames only (Eq. 3).  For the HMM topologies
 *    the paper names (a blank-like state per phone, Sec. 2) the blank is a
 *    set of units and a frame is blank when one of them exceeds the
 *    threshold; a lower frame rate decodes every frame_stride-th frame.
 *  - finalTransition then backtrace (Alg. 1): add final costs, take the best
 *    state, follow back-pointers.
 *  - Exact lattices (Sec. 1, Sec. 3): arcs between surviving tokens whose
 *    own prefix cost survives the destination's cutoff, then pruned to those
 *    whose best complete path lies within lattice_beam of the best path.
 *
 * Everything is float32 with no contraction (built with -ffp-contract=off).
 *
 * Parity unpinned: the paper fixes none of these conventions, so nothing
 * outside this file and the decoder pins them: the arc-index tie-break of
 * recombination, the lowest-state tie-break of the final argmin, the
 * fall-back to "every state final" when no final state is reached, and the
 * exact raw-lattice arc criterion (the kept set is pinned against brute
 * force only on dyadic inputs, where float32 arithmetic is exact).
 */
#include "oracle_wfst.h"

#include <float.h>
#include <math.h>
#include <stdlib.h>
#include <string.h>
#include <time.h>

#define EMPTY_TOK UINT64_MAX

/* ---------------------------------------------------------------------- */
/* ordered keys                                                            */
/* ---------------------------------------------------------------------- */

/* Map float32 to uint32 so that unsigned order equals numeric order (-0
 * sorts just below +0). */
static uint32_t okey(float x)
{
    uint32_t u;
    memcpy(&u, &x, 4);
    return (u >> 31) ? ~u : (u | 0x80000000u);
}

static float okey_value(uint32_t k)
{
    uint32_t u = (k >> 31) ? (k & 0x7fffffffu) : ~k;
    float x;
    memcpy(&x, &u, 4);
    return x;
}

static uint32_t fbits(float x)
{
    uint32_t u;
    memcpy(&u, &x, 4);
    return u;
}

/* A token: cost key in the high word, (arc index + 1) in the low word, so
 * that the unsigned minimum is the cheapest token with the lowest arc. */
static uint64_t make_tok(float cost, int64_t arc)
{
    return ((uint64_t)okey(cost) << 32) | (uint32_t)(arc + 1);
}

static float tok_cost(uint64_t t) { return okey_value((uint32_t)(t >> 32)); }
static int32_t tok_arc(uint64_t t) { return (int32_t)(uint32_t)t - 1; }

static double now_s(void)
{
    struct timespec ts;
    clock_gettime(CLOCK_MONOTONIC, &ts);
    return (double)ts.tv_sec + 1e-9 * (double)ts.tv_nsec;
}

/* ---------------------------------------------------------------------- */
/* growable arrays                                                         */
/* ---------------------------------------------------------------------- */

typedef struct { void *p; int64_t n, cap; size_t esz; } vec;

static int vec_push(vec *v, const void *x)
{
    if (v->n == v->cap) {
        int64_t nc = v->cap ? 2 * v->cap : 1024;
        void *q = realloc(v->p, (size_t)nc * v->esz);
        if (!q) return -1;
        v->p = q;
        v->cap = nc;
    }
    memcpy((char *)v->p + (size_t)v->n * v->esz, x, v->esz);
    v->n++;
    return 0;
}

/* ---------------------------------------------------------------------- */
/* validation                                                              */
/* ---------------------------------------------------------------------- */

int oracle_validate_graph(int32_t n, int64_t e, const int32_t *src, const int32_t *dst,
                          const int32_t *ilabel, const int32_t *olabel, const float *weight,
                          int32_t start, const float *final_weight)
{
    if (n < 1 || e < 0 || e >= 2147483647LL) return ORACLE_EINVAL;
    if (start < 0 || start >= n) return ORACLE_EINVAL;
    if (e > 0 && (!src || !dst || !ilabel || !olabel || !weight)) return ORACLE_EINVAL;
    for (int64_t a = 0; a < e; a++) {
        if (src[a] < 0 || src[a] >= n) return ORACLE_EINVAL;
        if (a > 0 && src[a] < src[a - 1]) return ORACLE_EINVAL;
        if (dst[a] < 0 || dst[a] >= n) return ORACLE_EINVAL;
        if (ilabel[a] < 0 || olabel[a] < 0) return ORACLE_EINVAL;
        if (!isfinite(weight[a])) return ORACLE_EINVAL;
        if (ilabel[a] == 0 && weight[a] < 0.0f) return ORACLE_EINVAL;
    }
    if (final_weight) {
        for (int32_t s = 0; s < n; s++) {
            if (isnan(final_weight[s])) return ORACLE_EINVAL;
            if (isinf(final_weight[s]) && final_weight[s] < 0) return ORACLE_EINVAL;
        }
    }
    /* epsilon subgraph must be acyclic: Kahn's algorithm */
    int32_t *indeg = calloc((size_t)n, sizeof(int32_t));
    int64_t *row = calloc((size_t)n + 1, sizeof(int64_t));
    int32_t *q = malloc((size_t)n * sizeof(int32_t));
    if (!indeg || !row || !q) { free(indeg); free(row); free(q); return ORACLE_ENOMEM; }
    for (int64_t a = 0; a < e; a++) row[src[a] + 1]++;
    for (int32_t s = 0; s < n; s++) row[s + 1] += row[s];
    for (int64_t a = 0; a < e; a++)
        if (ilabel[a] == 0) indeg[dst[a]]++;
    int64_t qh = 0, qt = 0;
    for (int32_t s = 0; s < n; s++)
        if (indeg[s] == 0) q[qt++] = s;
    while (qh < qt) {
        int32_t s = q[qh++];
        for (int64_t a = row[s]; a < row[s + 1]; a++)
            if (ilabel[a] == 0 && --indeg[dst[a]] == 0) q[qt++] = dst[a];
    }
    int ok = (qt == n);
    free(indeg); free(row); free(q);
    return ok ? ORACLE_OK : ORACLE_EINVAL;
}

/* ---------------------------------------------------------------------- */
/* the decoder                                                             */
/* ---------------------------------------------------------------------- */

typedef struct {
    int32_t n;
    int64_t e;
    const int32_t *src, *dst, *il;
    const float *w;
    int64_t *row;            /* arcs of state s: [row[s], row[s+1]) in user order */
} graph_t;

typedef struct {
    uint64_t *C;             /* token of every state in the current set, EMPTY if none */
    int32_t *reached;        /* states with a token in C */
    int64_t nreached;
    int32_t *queue;          /* FIFO ring for the epsilon closure */
    char *inq;
} work_t;

typedef struct { int32_t state; uint64_t tok; } surv_t;

typedef struct { int32_t frame, arc, kind; float p; int32_t gs, gd; float ex; } rec_t;

/* Lower C[d] to v if v is smaller; returns 1 when it did. */
static int touch(work_t *w, int32_t d, uint64_t v)
{
    if (v < w->C[d]) {
        if (w->C[d] == EMPTY_TOK) w->reached[w->nreached++] = d;
        w->C[d] = v;
        return 1;
    }
    return 0;
}

/* Epsilon closure: relax epsilon arcs from every reached state until no
 * token changes (FIFO order; the acyclic epsilon graph makes the fixed point
 * unique, so the order does not matter). */
static void closure(const graph_t *g, work_t *w)
{
    int64_t cap = (int64_t)g->n + 1, head = 0, tail = 0;
    for (int64_t i = 0; i < w->nreached; i++) {
        int32_t s = w->reached[i];
        w->queue[tail] = s; tail = (tail + 1) % cap; w->inq[s] = 1;
    }
    while (head != tail) {
        int32_t s = w->queue[head];
        head = (head + 1) % cap;
        w->inq[s] = 0;
        float c = tok_cost(w->C[s]);
        for (int64_t a = g->row[s]; a < g->row[s + 1]; a++) {
            if (g->il[a] != 0) continue;
            float cand = c + g->w[a];
            int32_t d = g->dst[a];
            if (touch(w, d, make_tok(cand, a)) && !w->inq[d]) {
                w->queue[tail] = d; tail = (tail + 1) % cap; w->inq[d] = 1;
            }
        }
    }
}

static int cmp_u32(const void *x, const void *y)
{
    uint32_t a = *(const uint32_t *)x, b = *(const uint32_t *)y;
    return (a > b) - (a < b);
}

static int cmp_surv(const void *x, const void *y)
{
    int32_t a = ((const surv_t *)x)->state, b = ((const surv_t *)y)->state;
    return (a > b) - (a < b);
}

static int cmp_rec(const void *x, const void *y)
{
    const rec_t *a = x, *b = y;
    if (a->frame != b->frame) return (a->frame > b->frame) - (a->frame < b->frame);
    return (a->arc > b->arc) - (a->arc < b->arc);
}

/* Beam + max-active pruning of the reached set.  Survivors (sorted by state)
 * are appended to *sv; returns their number, and the cutoff key in *cut. */
static int64_t prune(work_t *w, float beam, int32_t max_active, vec *sv, uint32_t *cut,
                     uint32_t *scratch)
{
    if (w->nreached == 0) { *cut = 0; return 0; }
    uint32_t b = UINT32_MAX;
    for (int64_t i = 0; i < w->nreached; i++) {
        uint32_t k = (uint32_t)(w->C[w->reached[i]] >> 32);
        if (k < b) b = k;
    }
    float cb = okey_value(b) + beam;
    uint32_t lim = okey(cb);
    if (lim > okey(FLT_MAX)) lim = okey(FLT_MAX);   /* infinite costs never survive */
    int64_t nk = 0;
    for (int64_t i = 0; i < w->nreached; i++) {
        uint32_t k = (uint32_t)(w->C[w->reached[i]] >> 32);
        if (k <= lim) scratch[nk++] = k;
    }
    uint32_t c = lim;
    if (max_active > 0 && nk > max_active) {
        qsort(scratch, (size_t)nk, sizeof(uint32_t), cmp_u32);
        uint32_t theta = scratch[max_active - 1];
        if (theta < c) c = theta;
    }
    int64_t first = sv->n;
    for (int64_t i = 0; i < w->nreached; i++) {
        int32_t s = w->reached[i];
        if ((uint32_t)(w->C[s] >> 32) <= c) {
            surv_t x = { s, w->C[s] };
            if (vec_push(sv, &x)) return -1;
        }
    }
    qsort((surv_t *)sv->p + first, (size_t)(sv->n - first), sizeof(surv_t), cmp_surv);
    *cut = c;
    return sv->n - first;
}

/* Index of state s in the sorted token set [lo, hi) of sv, or -1. */
static int64_t find_tok(const surv_t *sv, int64_t lo, int64_t hi, int32_t s)
{
    int64_t a = lo, b = hi;
    while (a < b) {
        int64_t mid = a + (b - a) / 2;
        if (sv[mid].state < s) a = mid + 1;
        else b = mid;
    }
    return (a < hi && sv[a].state == s) ? a : -1;
}

static void clear_reached(work_t *w)
{
    for (int64_t i = 0; i < w->nreached; i++) w->C[w->reached[i]] = EMPTY_TOK;
    w->nreached = 0;
}

static float fmin_key(float a, float b) { return okey(b) < okey(a) ? b : a; }

oracle_result *oracle_decode(int32_t n, int64_t e, const int32_t *src, const int32_t *dst,
                             const int32_t *ilabel, const int32_t *olabel, const float *weight,
                             int32_t start, const float *final_weight, const float *ll,
                             int32_t T, int32_t L, float beam, int32_t max_active,
                             float lattice_beam, float blank_threshold, int32_t blank_id)
{
    return oracle_decode_ext(n, e, src, dst, ilabel, olabel, weight, start, final_weight, ll, T, L, beam,
                             max_active, lattice_beam, blank_threshold, &blank_id, 1, 1);
}

oracle_result *oracle_decode_ext(int32_t n, int64_t e, const int32_t *src, const int32_t *dst,
                                 const int32_t *ilabel, const int32_t *olabel, const float *weight,
                                 int32_t start, const float *final_weight, const float *ll,
                                 int32_t T, int32_t L, float beam, int32_t max_active,
                                 float lattice_beam, float blank_threshold,
                                 const int32_t *blank_ids, int32_t nb, int32_t stride)
{
    oracle_result *r = calloc(1, sizeof(oracle_result));
    if (!r) return NULL;
    r->status = oracle_validate_graph(n, e, src, dst, ilabel, olabel, weight, start, final_weight);
    if (r->status != ORACLE_OK) return r;
    int32_t max_il = 0;
    for (int64_t a = 0; a < e; a++) if (ilabel[a] > max_il) max_il = ilabel[a];
    int bad_ids = nb < 1 || !blank_ids;
    for (int32_t i = 0; !bad_ids && i < nb; i++) bad_ids = blank_ids[i] < 0 || blank_ids[i] >= L;
    if (T < 0 || L < 1 || max_il > L || bad_ids || stride < 1 || !(beam > 0.0f) ||
        isnan(lattice_beam) || !(blank_threshold > 0.0f) || (T > 0 && !ll)) {
        r->status = ORACLE_EINVAL;
        return r;
    }
    const int lattice = lattice_beam >= 0.0f;

    graph_t g = { n, e, src, dst, ilabel, weight, calloc((size_t)n + 1, sizeof(int64_t)) };
    work_t w = { malloc((size_t)n * 8), malloc((size_t)n * 4), 0, malloc(((size_t)n + 1) * 4),
                 calloc((size_t)n, 1) };
    uint32_t *scratch = malloc((size_t)n * 4);
    vec sv = { NULL, 0, 0, sizeof(surv_t) };
    vec recs = { NULL, 0, 0, sizeof(rec_t) };
    int64_t *tok_off = malloc(((size_t)T + 2) * sizeof(int64_t));
    /* lattice records of frame j: emitting [eb[j], ee[j]), epsilon [xb[j], xe[j]) */
    int64_t *eb = calloc((size_t)T + 2, sizeof(int64_t)), *ee = calloc((size_t)T + 2, sizeof(int64_t));
    int64_t *xb = calloc((size_t)T + 2, sizeof(int64_t)), *xe = calloc((size_t)T + 2, sizeof(int64_t));
    uint32_t *cuts = malloc(((size_t)T + 1) * 4);
    int32_t *kept = malloc(((size_t)T + 1) * 4);
    float *e_node = NULL, *tot = NULL;
    if (!g.row || !w.C || !w.reached || !w.queue || !w.inq || !scratch || !tok_off || !eb ||
        !ee || !xb || !xe || !cuts || !kept) {
        r->status = ORACLE_ENOMEM;
        goto done;
    }
    for (int64_t a = 0; a < e; a++) g.row[src[a] + 1]++;
    for (int32_t s = 0; s < n; s++) g.row[s + 1] += g.row[s];
    for (int32_t s = 0; s < n; s++) w.C[s] = EMPTY_TOK;

    double t0 = now_s();

    /* isBlankFrame (Sec. 2, Alg. 1): U = {u : y_blank^u > threshold}, compared
     * in the log domain against one float32 threshold; a threshold above 1
     * makes no frame blank (frame-synchronous decoding).  With several
     * blank-like units a frame is blank when any of them passes; with a
     * frame stride only every stride-th frame is a candidate. */
    float thr = blank_threshold > 1.0f ? INFINITY : (float)log((double)blank_threshold);
    int32_t Tp = 0;
    for (int32_t t = 0; t < T; t += stride) {
        int blank = 0;
        for (int32_t i = 0; i < nb; i++)
            if (ll[(int64_t)t * L + blank_ids[i]] > thr) blank = 1;
        if (!blank) kept[Tp++] = t;
    }

    /* token set 0: the start token and its epsilon closure */
    touch(&w, start, make_tok(0.0f, -1));
    closure(&g, &w);
    tok_off[0] = 0;
    int64_t ns = prune(&w, beam, max_active, &sv, &cuts[0], scratch);
    if (ns < 0) { r->status = ORACLE_ENOMEM; goto done; }
    if (ns == 0) { r->status = ORACLE_ENOPATH; goto done; }
    tok_off[1] = sv.n;

    for (int32_t j = 0; j <= Tp; j++) {
        surv_t *S = (surv_t *)sv.p;
        int64_t lo = tok_off[j], hi = tok_off[j + 1];
        /* epsilon lattice arcs inside token set j */
        xb[j] = recs.n;
        if (lattice) {
            for (int64_t i = lo; i < hi; i++) {
                int32_t s = S[i].state;
                float c = tok_cost(S[i].tok);
                for (int64_t a = g.row[s]; a < g.row[s + 1]; a++) {
                    if (ilabel[a] != 0) continue;
                    float p = c + weight[a];
                    if (okey(p) > cuts[j]) continue;
                    int64_t gd = find_tok(S, lo, hi, dst[a]);
                    if (gd < 0) continue;
                    rec_t x = { j, (int32_t)a, 1, p, (int32_t)i, (int32_t)gd, INFINITY };
                    if (vec_push(&recs, &x)) { r->status = ORACLE_ENOMEM; goto done; }
                }
            }
        }
        xe[j] = recs.n;
        if (j == Tp) break;

        /* one frame of token passing (Alg. 1, ViterbiBeamSearch) */
        const float *row = ll + (int64_t)kept[j] * L;
        clear_reached(&w);
        for (int64_t i = lo; i < hi; i++) {
            int32_t s = S[i].state;
            float c = tok_cost(S[i].tok);
            for (int64_t a = g.row[s]; a < g.row[s + 1]; a++) {
                if (ilabel[a] == 0) continue;
                float t1 = c + weight[a];
                float cand = t1 - row[ilabel[a] - 1];
                touch(&w, dst[a], make_tok(cand, a));
                r->arcs_expanded++;
            }
        }
        closure(&g, &w);
        ns = prune(&w, beam, max_active, &sv, &cuts[j + 1], scratch);
        if (ns < 0) { r->status = ORACLE_ENOMEM; goto done; }
        if (ns == 0) { r->status = ORACLE_ENOPATH; goto done; }
        tok_off[j + 2] = sv.n;
        S = (surv_t *)sv.p;

        /* emitting lattice arcs from token set j to token set j+1 */
        eb[j] = recs.n;
        if (lattice) {
            int64_t lo2 = tok_off[j + 1], hi2 = tok_off[j + 2];
            for (int64_t i = lo; i < hi; i++) {
                int32_t s = S[i].state;
                float c = tok_cost(S[i].tok);
                for (int64_t a = g.row[s]; a < g.row[s + 1]; a++) {
                    if (ilabel[a] == 0) continue;
                    float t1 = c + weight[a];
                    float p = t1 - row[ilabel[a] - 1];
                    if (okey(p) > cuts[j + 1]) continue;
                    int64_t gd = find_tok(S, lo2, hi2, dst[a]);
                    if (gd < 0) continue;
                    rec_t x = { j, (int32_t)a, 0, p, (int32_t)i, (int32_t)gd, INFINITY };
                    if (vec_push(&recs, &x)) { r->status = ORACLE_ENOMEM; goto done; }
                }
            }
        }
        ee[j] = recs.n;
    }

    surv_t *S = (surv_t *)sv.p;
    int64_t ntok = sv.n;

    /* finalTransition (Alg. 1): add final costs on the last token set; if a
     * final-weight vector is given but no final state is active, fall back
     * to treating every state as final with cost 0. */
    int64_t lo = tok_off[Tp], hi = tok_off[Tp + 1];
    if (hi <= lo) { r->status = ORACLE_ENOPATH; goto done; }
    tot = malloc((size_t)(hi - lo) * sizeof(float));
    if (!tot) { r->status = ORACLE_ENOMEM; goto done; }
    int reached_final = 1, any = 0;
    for (int64_t i = lo; i < hi; i++) {
        float f = final_weight ? final_weight[S[i].state] : 0.0f;
        tot[i - lo] = tok_cost(S[i].tok) + f;
        if (okey(tot[i - lo]) < okey(INFINITY)) any = 1;
    }
    if (final_weight && !any) {
        reached_final = 0;
        for (int64_t i = lo; i < hi; i++) tot[i - lo] = tok_cost(S[i].tok) + 0.0f;
    }
    int64_t best = lo;
    for (int64_t i = lo; i < hi; i++)
        if (okey(tot[i - lo]) < okey(tot[best - lo])) best = i;   /* ties: lowest state */
    float B = tot[best - lo];
    if (!(okey(B) < okey(INFINITY))) { r->status = ORACLE_ENOPATH; goto done; }

    /* backtrace (Alg. 1) */
    {
        vec pa = { NULL, 0, 0, sizeof(int32_t) }, pf = { NULL, 0, 0, sizeof(int32_t) };
        int32_t j = Tp;
        int64_t i = best;
        for (int64_t guard = 0; guard <= ntok; guard++) {
            int32_t a = tok_arc(S[i].tok);
            if (a < 0) break;
            int32_t fr = -1;
            int32_t s = src[a];
            if (ilabel[a] != 0) {
                if (j == 0) { r->status = ORACLE_EINTERNAL; break; }
                fr = kept[j - 1];
                j--;
            }
            i = find_tok(S, tok_off[j], tok_off[j + 1], s);
            if (i < 0) { r->status = ORACLE_EINTERNAL; break; }
            vec_push(&pa, &a);
            vec_push(&pf, &fr);
        }
        if (r->status == ORACLE_OK) {
            int32_t *A = pa.p, *F = pf.p;
            for (int64_t k = 0; k < pa.n / 2; k++) {
                int32_t t = A[k]; A[k] = A[pa.n - 1 - k]; A[pa.n - 1 - k] = t;
                t = F[k]; F[k] = F[pa.n - 1 - k]; F[pa.n - 1 - k] = t;
            }
            r->path_len = (int32_t)pa.n;
            r->path_arcs = pa.p;
            r->path_frames = pf.p;
        } else {
            free(pa.p);
            free(pf.p);
            goto done;
        }
    }
    r->cost = B;
    r->final_state = S[best].state;
    r->reached_final = reached_final;

    /* lattice-beam pruning: backward extra costs.  e(T', s) = tot(s) - B;
     * an arc from (j, s) to (j', d) has ex = (p - c_j'(d)) + e(j', d);
     * e(j, s) is the minimum ex over the node's recorded out-arcs. */
    if (lattice) {
        rec_t *R = (rec_t *)recs.p;
        e_node = malloc((size_t)ntok * sizeof(float));
        if (!e_node && ntok) { r->status = ORACLE_ENOMEM; goto done; }
        for (int64_t i = 0; i < ntok; i++) e_node[i] = INFINITY;
        for (int64_t i = lo; i < hi; i++) e_node[i] = tot[i - lo] - B;
        for (int32_t j = Tp; j >= 0; j--) {
            if (j < Tp) {
                for (int64_t k = eb[j]; k < ee[j]; k++) {
                    float d1 = R[k].p - tok_cost(S[R[k].gd].tok);
                    R[k].ex = d1 + e_node[R[k].gd];
                    e_node[R[k].gs] = fmin_key(e_node[R[k].gs], R[k].ex);
                }
            }
            int changed = 1;
            while (changed) {
                changed = 0;
                for (int64_t k = xb[j]; k < xe[j]; k++) {
                    float d1 = R[k].p - tok_cost(S[R[k].gd].tok);
                    float ex = d1 + e_node[R[k].gd];
                    R[k].ex = ex;
                    if (okey(ex) < okey(e_node[R[k].gs])) { e_node[R[k].gs] = ex; changed = 1; }
                }
            }
        }
        r->lat_raw = recs.n;
        int64_t nk = 0;
        for (int64_t k = 0; k < recs.n; k++)
            if (R[k].ex <= lattice_beam) R[nk++] = R[k];
        qsort(R, (size_t)nk, sizeof(rec_t), cmp_rec);
        r->lat_n = nk;
        r->lat_frame = malloc((size_t)(nk ? nk : 1) * 4);
        r->lat_arc = malloc((size_t)(nk ? nk : 1) * 4);
        r->lat_cost = malloc((size_t)(nk ? nk : 1) * 4);
        r->lat_extra = malloc((size_t)(nk ? nk : 1) * 4);
        if (!r->lat_frame || !r->lat_arc || !r->lat_cost || !r->lat_extra) {
            r->status = ORACLE_ENOMEM;
            goto done;
        }
        for (int64_t k = 0; k < nk; k++) {
            r->lat_frame[k] = R[k].frame;
            r->lat_arc[k] = R[k].arc;
            r->lat_cost[k] = R[k].p;
            r->lat_extra[k] = R[k].ex;
        }
    }

    r->seconds = now_s() - t0;

    /* export token sets and counters */
    r->num_frames = T;
    r->num_decoded = Tp;
    r->kept = malloc(((size_t)Tp + 1) * 4);
    r->tok_off = malloc(((size_t)Tp + 2) * sizeof(int64_t));
    r->tok_state = malloc((size_t)(ntok ? ntok : 1) * 4);
    r->tok_cost_bits = malloc((size_t)(ntok ? ntok : 1) * 4);
    r->tok_arc = malloc((size_t)(ntok ? ntok : 1) * 4);
    r->cut_key = malloc(((size_t)Tp + 1) * 4);
    if (!r->kept || !r->tok_off || !r->tok_state || !r->tok_cost_bits || !r->tok_arc ||
        !r->cut_key) {
        r->status = ORACLE_ENOMEM;
        goto done;
    }
    memcpy(r->kept, kept, (size_t)Tp * 4);
    memcpy(r->tok_off, tok_off, ((size_t)Tp + 2) * sizeof(int64_t));
    memcpy(r->cut_key, cuts, ((size_t)Tp + 1) * 4);
    for (int64_t i = 0; i < ntok; i++) {
        r->tok_state[i] = S[i].state;
        r->tok_cost_bits[i] = fbits(tok_cost(S[i].tok));
        r->tok_arc[i] = tok_arc(S[i].tok);
        int32_t s = S[i].state;
        for (int64_t a = g.row[s]; a < g.row[s + 1]; a++)
            if (ilabel[a] == 0) r->eps_arcs++;
    }
    r->tokens = ntok;

done:
    free(g.row); free(w.C); free(w.reached); free(w.queue); free(w.inq); free(scratch);
    free(sv.p); free(recs.p); free(tok_off); free(eb); free(ee); free(xb); free(xe); free(cuts); free(kept);
    free(e_node); free(tot);
    return r;
}

void oracle_free(oracle_result *r)
{
    if (!r) return;
    free(r->path_arcs); free(r->path_frames); free(r->kept); free(r->tok_off);
    free(r->tok_state); free(r->tok_cost_bits); free(r->tok_arc); free(r->cut_key);
    free(r->lat_frame); free(r->lat_arc); free(r->lat_cost); free(r->lat_extra);
    free(r);
}
