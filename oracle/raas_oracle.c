/*
 * CPU oracle for page-based RaaS decode (TEST INFRASTRUCTURE ONLY).
 *
 * A plain, slow, fp64 reference of what the decode path computes, written
 * from the paper (arXiv 2502.11147): Algorithm 1 (RaaS Algorithm) for the
 * order of a decode step, Section 3.2 for the top-r / LRU timestamp rule and
 * prefill pinning, Section 3.3 for page granularity and the Quest-style
 * representative score. Only tests, the smoke check and the benchmark's CPU
 * baseline may call it; the product path never does. It shares no code with
 * the HIP path.
 *
 * One kvm (KV manager) holds the cache of one unit: one sequence, one layer,
 * one KV head, with the G query heads that share that KV head.
 *
 * Readings of points the paper leaves open (each is marked where it is used):
 *  R1 representative key: per-channel min and max of the page's keys, score
 *     = sum_c max(q_c*kmax_c, q_c*kmin_c), an upper bound on q.k for every key
 *     of the page (Quest's criterion, Section 3.3 adopts Quest's strategy).
 *  R2 GQA: one decision per unit; page score = max over the G query heads.
 *  R3 prefill longer than the budget: pin the first min(P_pages, S-1) pages
 *     and drop the rest (policy PIN_HEAD), or refuse (policy ERROR).
 *  R4 a partial last prefill page is not topped up by decode tokens.
 *  R5 a new page's timestamp is the clock at its creation; the clock is the
 *     token's absolute position.
 *  R6 ties of the oldest timestamp go to the smallest logical page id.
 *  R7 "top-r": n = #evictable pages, k = floor(r*n); the pages strictly above
 *     the (n-k)-th smallest score are refreshed (k = n: all; k = 0: none).
 *     Only decode (evictable) pages take part; the current tail page counts.
 *  R8 eviction is eager, in Algorithm 1's order: after the refresh, when the
 *     next token has no room (tail page full and no free slot).
 *  R9 softmax scale 1/sqrt(d); attention covers every resident token.
 *
 * Variants of R2 and R7 (off by default; orc_set_variant):
 *  aggregation 1: a page's score is the sum over the G query heads of that
 *     head's softmax probability over the ranked pages, the representative
 *     bound standing for the page's logit: sum_j exp(scale*(b_j(p) - M_j)) /
 *     sum_p' exp(scale*(b_j(p') - M_j)), M_j the head's largest bound,
 *     scale 1/sqrt(d). The paper names no such aggregation: the scale in
 *     particular is a reading, not a value the paper fixes. The pins hold
 *     the normalisation, a lone page's value, the G = 1 reduction to R2 and,
 *     through a step worked by hand (tests/golden), the scale the oracle
 *     uses: under scale 1 that step would refresh another page.
 *  rank_pinned 1: the pinned prompt pages are ranked together with the
 *     decode pages (n and k count them); only decode pages take timestamps.
 * Variant of the decision scope (orc_decode_group): one page table per
 *  (sequence, layer) shared by its KV heads, the page score aggregating all
 *  of the sequence's query heads.
 * Variant of R3 for long prompts (orc_set_prompt_selection), the combination
 *  the paper recommends for small budgets or long prompts (Section 4.2 and
 *  its Limitations): Quest on the prompt pages, RaaS on the decode pages.
 *  Readings (the paper gives no more than the recommendation): the prompt
 *  keeps its own region of prompt_slots slots (all its pages are stored, as
 *  Quest keeps every token), the decode pages live in the slots after it
 *  under RaaS as above, and each step attends to the prompt_topk prompt pages
 *  with the largest representative bound (max over the G heads, as R1/R2),
 *  ties to the lower slot, plus every decode page and the new token.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_OK 0
#define ORC_E_INVALID (-1)
#define ORC_E_BUDGET (-2)
#define ORC_E_STATE (-3)
#define ORC_E_INTERNAL (-10)

enum { FREE = 0, PINNED = 1, EVICTABLE = 2 };
enum { POLICY_PIN_HEAD = 0, POLICY_ERROR = 1 };

typedef struct {
    int G, d, ps, S, policy;
    int aggregation, rank_pinned; /* variants of R2 and R7, 0 by default */
    int decode_base, prompt_topk; /* prompt selection: first decode slot, pages attended (-1: off) */
    unsigned char* attend;        /* [S] slots the step attends to */
    double r;
    /* per page slot */
    int *state, *lid, *fill, *ts;
    double *K, *V;       /* [S][ps][d] */
    double *kmin, *kmax; /* [S][d] representative keys (R1) */
    /* per unit */
    int tail, next_lid, clock, prefilled;
    /* diagnostics of the last decode step */
    double *score; /* [S], NaN where the slot is not evictable */
    double theta;  /* the threshold; -inf when every page was refreshed, NaN when none */
    int n_evictable, k_refreshed, evicted;
    int evicted_slot, evicted_tail; /* slot of the evicted page, and whether it was the tail */
} orc_kvm;

orc_kvm* orc_new(int G, int d, int ps, int S, double r, int policy) {
    if (G < 1 || d < 1 || ps < 1 || S < 2 || !(r >= 0.0 && r <= 1.0)) return NULL;
    if (policy != POLICY_PIN_HEAD && policy != POLICY_ERROR) return NULL;
    orc_kvm* m = (orc_kvm*)calloc(1, sizeof(orc_kvm));
    m->G = G; m->d = d; m->ps = ps; m->S = S; m->r = r; m->policy = policy;
    m->state = (int*)calloc((size_t)S, sizeof(int));
    m->lid = (int*)calloc((size_t)S, sizeof(int));
    m->fill = (int*)calloc((size_t)S, sizeof(int));
    m->ts = (int*)calloc((size_t)S, sizeof(int));
    m->K = (double*)calloc((size_t)S * ps * d, sizeof(double));
    m->V = (double*)calloc((size_t)S * ps * d, sizeof(double));
    m->kmin = (double*)calloc((size_t)S * d, sizeof(double));
    m->kmax = (double*)calloc((size_t)S * d, sizeof(double));
    m->score = (double*)calloc((size_t)S, sizeof(double));
    m->attend = (unsigned char*)calloc((size_t)S, 1);
    m->prompt_topk = -1;
    for (int s = 0; s < S; ++s) {
        m->state[s] = FREE;
        m->lid[s] = -1;
        m->ts[s] = -1;
        m->score[s] = NAN;
    }
    m->tail = -1;
    m->evicted = -1;
    m->evicted_slot = -1;
    m->theta = NAN;
    return m;
}

int orc_set_variant(orc_kvm* m, int aggregation, int rank_pinned) {
    if (!m || aggregation < 0 || aggregation > 1 || rank_pinned < 0 || rank_pinned > 1) return ORC_E_INVALID;
    if (rank_pinned && m->prompt_topk >= 0) return ORC_E_INVALID;
    m->aggregation = aggregation;
    m->rank_pinned = rank_pinned;
    return ORC_OK;
}

/* Quest on the prompt pages (see the header): prompt_slots slots hold the
 * prompt, decode pages use the rest; each step attends to the topk prompt
 * pages of largest bound. Before the prefill only; not with rank_pinned. */
int orc_set_prompt_selection(orc_kvm* m, int prompt_slots, int topk) {
    if (!m || m->prefilled || m->rank_pinned) return ORC_E_INVALID;
    if (prompt_slots < 0 || prompt_slots > m->S - 1 || topk < 0) return ORC_E_INVALID;
    m->decode_base = prompt_slots;
    m->prompt_topk = topk;
    return ORC_OK;
}

void orc_free(orc_kvm* m) {
    if (!m) return;
    free(m->attend);
    free(m->state); free(m->lid); free(m->fill); free(m->ts);
    free(m->K); free(m->V); free(m->kmin); free(m->kmax); free(m->score);
    free(m);
}

static void page_reset_representative(orc_kvm* m, int s) {
    for (int c = 0; c < m->d; ++c) {
        m->kmin[(size_t)s * m->d + c] = INFINITY;
        m->kmax[(size_t)s * m->d + c] = -INFINITY;
    }
}

/* write one token into slot s at its next position and widen the page's
 * per-channel min/max (R1) */
static void page_store_token(orc_kvm* m, int s, const double* k, const double* v) {
    const int d = m->d;
    size_t off = ((size_t)s * m->ps + m->fill[s]) * d;
    for (int c = 0; c < d; ++c) {
        m->K[off + c] = k[c];
        m->V[off + c] = v[c];
        if (k[c] < m->kmin[(size_t)s * d + c]) m->kmin[(size_t)s * d + c] = k[c];
        if (k[c] > m->kmax[(size_t)s * d + c]) m->kmax[(size_t)s * d + c] = k[c];
    }
    m->fill[s] += 1;
}

/* The prefill stage of Algorithm 1's cache store: the prompt's K/V go into
 * pages that are never evicted (Section 3.1 keeps every prefill token).
 * K, V: [P][d]. */
int orc_prefill(orc_kvm* m, const double* K, const double* V, int P) {
    if (!m || P < 0 || (P > 0 && (!K || !V))) return ORC_E_INVALID;
    if (m->prefilled) return ORC_E_STATE;
    const int ps = m->ps;
    int pages = (P + ps - 1) / ps;
    int keep = pages;
    /* R3: at least one slot stays for decode pages; with prompt selection the
     * prompt has its own region */
    const int cap = m->prompt_topk >= 0 ? m->decode_base : m->S - 1;
    if (keep > cap) {
        if (m->policy == POLICY_ERROR) return ORC_E_BUDGET;
        keep = cap;
    }
    for (int p = 0; p < keep; ++p) {
        m->state[p] = PINNED;
        m->lid[p] = p;
        m->ts[p] = -1;
        m->fill[p] = 0;
        page_reset_representative(m, p);
        for (int t = p * ps; t < P && t < (p + 1) * ps; ++t)
            page_store_token(m, p, K + (size_t)t * m->d, V + (size_t)t * m->d);
    }
    m->next_lid = pages;
    m->tail = -1; /* R4: decode tokens start a fresh page */
    m->clock = P; /* R5 */
    m->prefilled = 1;
    return ORC_OK;
}

/* Algorithm 1's attention step: exact softmax attention of each of the G
 * queries over the cached tokens with the new one appended (R9).
 * out: [G][d]. */
static void attention(const orc_kvm* m, const double* q, const double* k_new, const double* v_new,
                      double* out) {
    const int G = m->G, d = m->d, ps = m->ps;
    const double scale = 1.0 / sqrt((double)d);
    int n_old = 0;
    for (int s = 0; s < m->S; ++s)
        if (m->attend[s]) n_old += m->fill[s];
    const int n = n_old + 1;
    double* Kc = (double*)malloc(sizeof(double) * (size_t)n * d);
    double* Vc = (double*)malloc(sizeof(double) * (size_t)n * d);
    double* logit = (double*)malloc(sizeof(double) * (size_t)n);
    int i = 0;
    for (int s = 0; s < m->S; ++s) { /* K_old, V_old */
        if (!m->attend[s]) continue;
        for (int t = 0; t < m->fill[s]; ++t, ++i) {
            memcpy(Kc + (size_t)i * d, m->K + ((size_t)s * ps + t) * d, sizeof(double) * d);
            memcpy(Vc + (size_t)i * d, m->V + ((size_t)s * ps + t) * d, sizeof(double) * d);
        }
    }
    memcpy(Kc + (size_t)i * d, k_new, sizeof(double) * d); /* :: K_new */
    memcpy(Vc + (size_t)i * d, v_new, sizeof(double) * d);
    for (int j = 0; j < G; ++j) {
        const double* qj = q + (size_t)j * d;
        double mx = -INFINITY;
        for (int t = 0; t < n; ++t) {
            double acc = 0.0;
            for (int c = 0; c < d; ++c) acc += qj[c] * Kc[(size_t)t * d + c];
            logit[t] = acc * scale;
            if (logit[t] > mx) mx = logit[t];
        }
        double den = 0.0;
        for (int c = 0; c < d; ++c) out[(size_t)j * d + c] = 0.0;
        for (int t = 0; t < n; ++t) {
            double p = exp(logit[t] - mx);
            den += p;
            for (int c = 0; c < d; ++c) out[(size_t)j * d + c] += p * Vc[(size_t)t * d + c];
        }
        for (int c = 0; c < d; ++c) out[(size_t)j * d + c] /= den;
    }
    free(Kc); free(Vc); free(logit);
}

static int cmp_double(const void* a, const void* b) {
    double x = *(const double*)a, y = *(const double*)b;
    return (x > y) - (x < y);
}

/* Algorithm 1's fullness test: the next token has no room (R8) */
static int is_full(const orc_kvm* m) {
    if (m->tail >= 0 && m->fill[m->tail] < m->ps) return 0;
    for (int s = m->decode_base; s < m->S; ++s)
        if (m->state[s] == FREE) return 0;
    return 1;
}

/* the slots a step attends to: every resident page, except that with prompt
 * selection only the prompt_topk pinned pages of largest bound (max over the
 * heads of sum_c max(q_c kmax_c, q_c kmin_c)) are taken, ties to the lower
 * slot */
static void select_attended(orc_kvm* m, const double* q) {
    const int S = m->S, G = m->G, d = m->d;
    int np = 0;
    for (int s = 0; s < S; ++s) {
        m->attend[s] = m->state[s] != FREE;
        np += m->state[s] == PINNED;
    }
    if (m->prompt_topk < 0 || np <= m->prompt_topk) return;
    double* b = (double*)malloc(sizeof(double) * (size_t)S);
    for (int s = 0; s < S; ++s) {
        if (m->state[s] != PINNED) continue;
        double best = -INFINITY;
        for (int j = 0; j < G; ++j) {
            double acc = 0.0;
            for (int c = 0; c < d; ++c) {
                const double x = q[(size_t)j * d + c] * m->kmax[(size_t)s * d + c];
                const double y = q[(size_t)j * d + c] * m->kmin[(size_t)s * d + c];
                acc += x > y ? x : y;
            }
            if (acc > best) best = acc;
        }
        b[s] = best;
    }
    for (int s = 0; s < S; ++s) {
        if (m->state[s] != PINNED) continue;
        int above = 0;
        for (int o = 0; o < S; ++o)
            if (m->state[o] == PINNED && (b[o] > b[s] || (b[o] == b[s] && o < s))) ++above;
        m->attend[s] = above < m->prompt_topk;
    }
    free(b);
}

/* The new token's K/V go into the tail page, or into a fresh page taken from
 * the lowest free slot when the tail is full or absent (Section 3.3). Without
 * k_new/v_new (retention-only runs) the token takes its place but no
 * payload. */
static int store_new_token(orc_kvm* m, const double* k_new, const double* v_new) {
    const int S = m->S, c = m->clock;
    if (m->tail < 0 || m->fill[m->tail] == m->ps) {
        int s = -1;
        for (int i = m->decode_base; i < S; ++i)
            if (m->state[i] == FREE) { s = i; break; }
        if (s < 0) return ORC_E_INTERNAL; /* eager eviction leaves a free slot */
        m->state[s] = EVICTABLE;
        m->lid[s] = m->next_lid++;
        m->fill[s] = 0;
        m->ts[s] = c; /* R5 */
        page_reset_representative(m, s);
        m->tail = s;
    }
    if (k_new && v_new) {
        page_store_token(m, m->tail, k_new, v_new);
    } else {
        m->fill[m->tail] += 1; /* retention-only run: no payload */
    }
    return ORC_OK;
}

/* the ranked pages: the decode pages, and the pinned ones too when
 * rank_pinned (R7) */
#define RANKED(st) ((st) == EVICTABLE || (m->rank_pinned && (st) == PINNED))

/* per-head bounds of the ranked pages (R1): for this unit's G query heads
 * j, bound[s*H + h0 + j] = sum_c max(q_jc*kmax_sc, q_jc*kmin_sc). */
static void head_bounds(const orc_kvm* m, const double* q, double* bound, int H, int h0) {
    const int G = m->G, d = m->d;
    for (int s = 0; s < m->S; ++s) {
        if (!RANKED(m->state[s])) continue;
        for (int j = 0; j < G; ++j) {
            double acc = 0.0;
            for (int ch = 0; ch < d; ++ch) {
                double a = q[(size_t)j * d + ch] * m->kmax[(size_t)s * d + ch];
                double b = q[(size_t)j * d + ch] * m->kmin[(size_t)s * d + ch];
                acc += (a > b) ? a : b;
            }
            bound[(size_t)s * H + h0 + j] = acc;
        }
    }
}

/* one score per ranked page from the bounds of H query heads (R2, or the
 * softmax variant); m->score is NaN elsewhere */
static void aggregate(orc_kvm* m, const double* bound, int H) {
    const int S = m->S;
    for (int s = 0; s < S; ++s) m->score[s] = NAN;
    if (m->aggregation == 0) { /* R2: max over the heads */
        for (int s = 0; s < S; ++s) {
            if (!RANKED(m->state[s])) continue;
            double best = -INFINITY;
            for (int j = 0; j < H; ++j)
                if (bound[(size_t)s * H + j] > best) best = bound[(size_t)s * H + j];
            m->score[s] = best;
        }
    } else { /* sum over the heads of each head's softmax over the ranked pages */
        const double scale = 1.0 / sqrt((double)m->d);
        for (int s = 0; s < S; ++s)
            if (RANKED(m->state[s])) m->score[s] = 0.0;
        for (int j = 0; j < H; ++j) {
            double mx = -INFINITY, z = 0.0;
            for (int s = 0; s < S; ++s)
                if (RANKED(m->state[s]) && bound[(size_t)s * H + j] > mx) mx = bound[(size_t)s * H + j];
            for (int s = 0; s < S; ++s)
                if (RANKED(m->state[s])) z += exp(scale * (bound[(size_t)s * H + j] - mx));
            for (int s = 0; s < S; ++s)
                if (RANKED(m->state[s])) m->score[s] += exp(scale * (bound[(size_t)s * H + j] - mx)) / z;
        }
    }
}

/* new timestamps (the clock c) to the decode pages among the top-r ranked
 * scores (R7) */
static void refresh(orc_kvm* m, int c) {
    const int S = m->S;
    int n = 0;
    for (int s = 0; s < S; ++s)
        if (RANKED(m->state[s])) ++n;
    int k = (int)floor(m->r * (double)n);
    m->n_evictable = n;
    m->k_refreshed = k;
    m->theta = NAN;
    if (k > 0) {
        double theta = -INFINITY;
        if (k < n) {
            double* sorted = (double*)malloc(sizeof(double) * (size_t)n);
            int i = 0;
            for (int s = 0; s < S; ++s)
                if (RANKED(m->state[s])) sorted[i++] = m->score[s];
            qsort(sorted, (size_t)n, sizeof(double), cmp_double);
            theta = sorted[n - k - 1]; /* the (n-k)-th smallest */
            free(sorted);
        }
        m->theta = theta;
        for (int s = 0; s < S; ++s)
            if (m->state[s] == EVICTABLE && m->score[s] > theta) m->ts[s] = c;
    }
}

/* Eviction when the cache is full: the evictable page of oldest timestamp
 * goes (R6, R8) */
static int evict_if_full(orc_kvm* m) {
    const int S = m->S;
    m->evicted = -1;
    m->evicted_slot = -1;
    m->evicted_tail = 0;
    if (is_full(m)) {
        int v = -1;
        for (int s = 0; s < S; ++s) {
            if (m->state[s] != EVICTABLE) continue;
            if (v < 0 || m->ts[s] < m->ts[v] || (m->ts[s] == m->ts[v] && m->lid[s] < m->lid[v])) v = s;
        }
        if (v < 0) return ORC_E_INTERNAL;
        m->evicted = m->lid[v];
        m->evicted_slot = v;
        m->evicted_tail = m->tail == v;
        m->state[v] = FREE;
        m->lid[v] = -1;
        m->ts[v] = -1;
        m->fill[v] = 0;
        if (m->tail == v) m->tail = -1;
    }
    return ORC_OK;
}

/*
 * One decode step of one unit: attention, then the decode stage of the
 * cache store: the new token joins the cache, the top-r pages are stamped
 * with the current clock, and a full cache evicts its page of oldest stamp
 * (Algorithm 1, Section 3.3).
 *
 * q: [G][d]; k_new, v_new: [d]; out: [G][d] or NULL (attention skipped).
 * injected: NULL, or per-slot page scores that replace the representative
 * scores (used to drive the retention policy directly in tests).
 */
int orc_decode(orc_kvm* m, const double* q, const double* k_new, const double* v_new, double* out,
               const double* injected) {
    if (!m) return ORC_E_INVALID;
    if (!m->prefilled) return ORC_E_STATE;
    if (!injected && (!q || !k_new || !v_new)) return ORC_E_INVALID;
    const int G = m->G, S = m->S;
    const int c = m->clock;

    if (out) {
        select_attended(m, q);
        attention(m, q, k_new, v_new, out);
    }
    int rc = store_new_token(m, k_new, v_new);
    if (rc != ORC_OK) return rc;

    if (injected) {
        for (int s = 0; s < S; ++s) m->score[s] = RANKED(m->state[s]) ? injected[s] : NAN;
    } else {
        double* bound = (double*)malloc(sizeof(double) * (size_t)S * G);
        head_bounds(m, q, bound, G, 0);
        aggregate(m, bound, G);
        free(bound);
    }
    refresh(m, c);
    rc = evict_if_full(m);
    if (rc != ORC_OK) return rc;
    m->clock = c + 1;
    return ORC_OK;
}
#undef RANKED

/*
 * Variant of R2 with one decision per (sequence, layer): one decode step of
 * a sequence whose n KV heads share one page table. ms[h] holds KV head h
 * with its G query heads; every unit attends over its own keys and stores
 * its own new token, and a page's score aggregates the bounds of all n*G
 * query heads (the max, or the sum of per-head softmax), each head against
 * its own KV head's representative key. The refresh and eviction are then
 * the same for every KV head. The n units must be alike (configuration,
 * prefill length, steps), so their slot states are identical.
 * q: [n][G][d]; k_new, v_new: [n][d]; out: [n][G][d] or NULL.
 */
int orc_decode_group(orc_kvm** ms, int n, const double* q, const double* k_new, const double* v_new,
                     double* out) {
    if (!ms || n < 1 || !q || !k_new || !v_new) return ORC_E_INVALID;
    const orc_kvm* a = ms[0];
    for (int h = 0; h < n; ++h) {
        const orc_kvm* b = ms[h];
        if (!b) return ORC_E_INVALID;
        if (!b->prefilled) return ORC_E_STATE;
        if (b->G != a->G || b->d != a->d || b->ps != a->ps || b->S != a->S || b->r != a->r ||
            b->aggregation != a->aggregation || b->rank_pinned != a->rank_pinned ||
            b->decode_base != a->decode_base || b->prompt_topk != a->prompt_topk ||
            b->clock != a->clock || b->tail != a->tail || b->next_lid != a->next_lid)
            return ORC_E_INVALID;
        for (int s = 0; s < a->S; ++s)
            if (b->state[s] != a->state[s] || b->lid[s] != a->lid[s] || b->ts[s] != a->ts[s] ||
                b->fill[s] != a->fill[s])
                return ORC_E_INVALID;
    }
    const int G = a->G, d = a->d, S = a->S, H = n * G;
    const int c = a->clock;
    for (int h = 0; h < n; ++h) {
        if (out) {
            select_attended(ms[h], q + (size_t)h * G * d);
            attention(ms[h], q + (size_t)h * G * d, k_new + (size_t)h * d, v_new + (size_t)h * d,
                      out + (size_t)h * G * d);
        }
        int rc = store_new_token(ms[h], k_new + (size_t)h * d, v_new + (size_t)h * d);
        if (rc != ORC_OK) return rc;
    }
    double* bound = (double*)malloc(sizeof(double) * (size_t)S * H);
    for (int h = 0; h < n; ++h) head_bounds(ms[h], q + (size_t)h * G * d, bound, H, h * G);
    aggregate(ms[0], bound, H);
    free(bound);
    for (int h = 0; h < n; ++h) {
        if (h > 0) memcpy(ms[h]->score, ms[0]->score, sizeof(double) * (size_t)S);
        refresh(ms[h], c);
        int rc = evict_if_full(ms[h]);
        if (rc != ORC_OK) return rc;
        ms[h]->clock = c + 1;
    }
    return ORC_OK;
}

/* page table (lid or -1), timestamps (-1 for pinned and free), state, fill */
void orc_state(const orc_kvm* m, int* page_table, int* ts, int* state, int* fill, int* unit) {
    for (int s = 0; s < m->S; ++s) {
        if (page_table) page_table[s] = (m->state[s] == FREE) ? -1 : m->lid[s];
        if (ts) ts[s] = (m->state[s] == EVICTABLE) ? m->ts[s] : -1;
        if (state) state[s] = m->state[s];
        if (fill) fill[s] = m->fill[s];
    }
    if (unit) {
        unit[0] = m->tail;
        unit[1] = m->next_lid;
        unit[2] = m->clock;
        unit[3] = m->evicted;
        unit[4] = m->n_evictable;
        unit[5] = m->k_refreshed;
    }
}

/*
 * Test hook of the lockstep comparison (not part of the method): after a
 * step whose threshold was a near tie, take another implementation's
 * retention decision for this step, given as its page table (lid or -1 per
 * slot), timestamps (-1 unless evictable) and evicted lid. Only what the
 * step itself decided may differ from this kvm's state: the timestamps of
 * evictable pages and which full page was evicted. The page this kvm
 * evicted comes back from its slot (its keys and values are still there:
 * nothing is stored between the eviction and the next step), and the page
 * the other side evicted is freed. Anything else is ORC_E_INVALID and
 * leaves the state unchanged.
 */
int orc_adopt_retention(orc_kvm* m, const int* page_table, const int* ts, int evicted) {
    if (!m || !page_table || !ts || !m->prefilled) return ORC_E_INVALID;
    const int S = m->S;
    int freed = -1, back = -1;
    for (int s = 0; s < S; ++s) {
        const int pt = page_table[s];
        if (m->state[s] == PINNED) {
            if (pt != m->lid[s] || ts[s] != -1) return ORC_E_INVALID;
        } else if (m->state[s] == EVICTABLE) {
            if (pt == m->lid[s]) {
                if (ts[s] < 0 || ts[s] > m->clock) return ORC_E_INVALID;
            } else if (pt == -1 && ts[s] == -1 && m->fill[s] == m->ps && freed < 0 && evicted == m->lid[s]) {
                freed = s; /* the other side's victim: a full page */
            } else {
                return ORC_E_INVALID;
            }
        } else { /* FREE */
            if (pt == -1) {
                if (ts[s] != -1) return ORC_E_INVALID;
            } else if (s == m->evicted_slot && pt == m->evicted && ts[s] >= 0 && ts[s] <= m->clock) {
                back = s; /* this kvm's victim, kept by the other side */
            } else {
                return ORC_E_INVALID;
            }
        }
    }
    if ((freed >= 0) != (back >= 0)) return ORC_E_INVALID; /* one eviction each, or the same one */
    if (freed < 0 && evicted != m->evicted) return ORC_E_INVALID;
    for (int s = 0; s < S; ++s)
        if (m->state[s] == EVICTABLE && s != freed) m->ts[s] = ts[s];
    if (back >= 0) {
        m->state[back] = EVICTABLE;
        m->lid[back] = m->evicted;
        m->fill[back] = m->ps; /* evicted pages are full */
        m->ts[back] = ts[back];
        if (m->evicted_tail) m->tail = back;
        m->state[freed] = FREE;
        m->lid[freed] = -1;
        m->ts[freed] = -1;
        m->fill[freed] = 0;
        m->evicted_tail = m->tail == freed;
        if (m->tail == freed) m->tail = -1;
        m->evicted = evicted;
        m->evicted_slot = freed;
    }
    return ORC_OK;
}

/* orc_state of n kvms at once: page_table, ts [n][S] (S of the first), evicted [n] */
void orc_state_batch(orc_kvm** ms, int n, int* page_table, int* ts, int* evicted) {
    const int S = ms[0]->S;
    for (int u = 0; u < n; ++u) {
        orc_state(ms[u], page_table + (size_t)u * S, ts + (size_t)u * S, NULL, NULL, NULL);
        evicted[u] = ms[u]->evicted;
    }
}

/* orc_last_scores of n kvms at once: score [n][S], theta [n] */
void orc_scores_batch(orc_kvm** ms, int n, double* score, double* theta) {
    const int S = ms[0]->S;
    for (int u = 0; u < n; ++u) {
        memcpy(score + (size_t)u * S, ms[u]->score, sizeof(double) * (size_t)S);
        theta[u] = ms[u]->theta;
    }
}

/* the slots the last step attended to (1) or not (0) */
void orc_last_attended(const orc_kvm* m, int* out) {
    for (int s = 0; s < m->S; ++s) out[s] = m->attend[s];
}

/* per-slot scores of the last step (NaN where not evictable) and the threshold */
void orc_last_scores(const orc_kvm* m, double* score, double* theta) {
    if (score) memcpy(score, m->score, sizeof(double) * (size_t)m->S);
    if (theta) *theta = m->theta;
}

/* the resident keys / values in slot order, for tests: [S][ps][d] */
void orc_pages(const orc_kvm* m, double* K, double* V, double* kmin, double* kmax) {
    size_t n = (size_t)m->S * m->ps * m->d;
    if (K) memcpy(K, m->K, sizeof(double) * n);
    if (V) memcpy(V, m->V, sizeof(double) * n);
    if (kmin) memcpy(kmin, m->kmin, sizeof(double) * (size_t)m->S * m->d);
    if (kmax) memcpy(kmax, m->kmax, sizeof(double) * (size_t)m->S * m->d);
}

/*
 * One decode step for n independent units (OpenMP across units only). The
 * inputs are float32 (values of the workload's dtype, widened exactly).
 * q: [n][G][d]; k, v: [n][d]; out: [n][G][d] fp64 or NULL.
 */
int orc_decode_batch(orc_kvm** ms, int n, const float* q, const float* k, const float* v,
                     double* out) {
    int status = ORC_OK;
#pragma omp parallel for schedule(dynamic, 1)
    for (int u = 0; u < n; ++u) {
        orc_kvm* m = ms[u];
        const int G = m->G, d = m->d;
        double* qd = (double*)malloc(sizeof(double) * (size_t)(G + 2) * d);
        double* kd = qd + (size_t)G * d;
        double* vd = kd + d;
        for (int i = 0; i < G * d; ++i) qd[i] = (double)q[(size_t)u * G * d + i];
        for (int i = 0; i < d; ++i) {
            kd[i] = (double)k[(size_t)u * d + i];
            vd[i] = (double)v[(size_t)u * d + i];
        }
        int rc = orc_decode(m, qd, kd, vd, out ? out + (size_t)u * G * d : NULL, NULL);
        if (rc != ORC_OK) {
#pragma omp critical
            status = rc;
        }
        free(qd);
    }
    return status;
}

void orc_set_threads(int n) {
#ifdef _OPENMP
    extern void omp_set_num_threads(int);
    if (n >= 1) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

int orc_threads(void) {
#ifdef _OPENMP
    extern int omp_get_max_threads(void);
    return omp_get_max_threads();
#else
    return 1;
#endif
}
