/*
 * Memory and undefined-behaviour check of the CPU oracle and the input
 * generator (test infrastructure): this driver is linked with
 * oracle/raas_oracle.c and synth/raas_synth.c under AddressSanitizer and
 * UndefinedBehaviorSanitizer (gcc -fsanitize=address,undefined, recovery
 * off) by tests/test_sanitize.py, and drives every entry point through the
 * configurations the tests use: the default rule and its variants, small
 * and large slot counts, prompts over the budget, Quest on the prompt, the
 * grouped (one page table per sequence) step, retention-only steps with
 * injected scores, the batched calls and the lockstep adopt hook. Any
 * sanitizer report ends the process with a nonzero status.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

typedef struct orc_kvm orc_kvm;
orc_kvm* orc_new(int G, int d, int ps, int S, double r, int policy);
int orc_set_variant(orc_kvm* m, int aggregation, int rank_pinned);
int orc_set_prompt_selection(orc_kvm* m, int prompt_slots, int topk);
void orc_free(orc_kvm* m);
int orc_prefill(orc_kvm* m, const double* K, const double* V, int P);
int orc_decode(orc_kvm* m, const double* q, const double* k_new, const double* v_new, double* out,
               const double* injected);
int orc_decode_group(orc_kvm** ms, int n, const double* q, const double* k_new, const double* v_new, double* out);
void orc_state(const orc_kvm* m, int* page_table, int* ts, int* state, int* fill, int* unit);
int orc_adopt_retention(orc_kvm* m, const int* page_table, const int* ts, int evicted);
void orc_state_batch(orc_kvm** ms, int n, int* page_table, int* ts, int* evicted);
void orc_scores_batch(orc_kvm** ms, int n, double* score, double* theta);
void orc_last_attended(const orc_kvm* m, int* out);
void orc_last_scores(const orc_kvm* m, double* score, double* theta);
void orc_pages(const orc_kvm* m, double* K, double* V, double* kmin, double* kmax);
int orc_decode_batch(orc_kvm** ms, int n, const float* q, const float* k, const float* v, double* out);

typedef struct {
    int32_t batch, n_layers, n_q_heads, n_kv_heads, head_dim;
    int32_t prefill_len;
    int32_t dtype;
    int32_t ms_period;
    int32_t ms_phase_random;
    int32_t ms_wmin, ms_wmax;
    double outlier_p;
    uint64_t seed;
} synth_workload;
void synth_prefill(const synth_workload* w, int layer, float* K, float* V);
void synth_prefill_units(const synth_workload* w, int layer, const int* units, int nu, float* K, float* V);
int synth_active_milestones(const synth_workload* w, int layer, int seq, int kvh, int t, int* steps, int cap);
void synth_steps(const synth_workload* w, int layer, int t0, int n, float* q, float* k, float* v);
void synth_steps_units(const synth_workload* w, int layer, int t0, int n, const int* units, int nu, float* q,
                       float* k, float* v);
void synth_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]);

#define CHECK(x)                                                            \
    do {                                                                    \
        if (!(x)) {                                                         \
            fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #x); \
            exit(2);                                                        \
        }                                                                   \
    } while (0)

static double* widen(const float* x, size_t n) {
    double* y = (double*)malloc(sizeof(double) * (n ? n : 1));
    for (size_t i = 0; i < n; ++i) y[i] = x[i];
    return y;
}

/* One configuration: B sequences of H KV heads (G query heads each), its
 * own seeded inputs, T decode steps through every entry point. */
static void run_case(int B, int H, int G, int d, int ps, int S, int P, int T, double r, int agg, int rank_pinned,
                     int prompt_slots, int topk, int grouped, double outlier_p) {
    synth_workload w = {B, 1, H * G, H, d, P, 1, 16, 1, 8, 64, outlier_p, 12345u};
    const int U = B * H;
    float* Kp = (float*)malloc(sizeof(float) * (size_t)U * (P ? P : 1) * d);
    float* Vp = (float*)malloc(sizeof(float) * (size_t)U * (P ? P : 1) * d);
    synth_prefill(&w, 0, Kp, Vp);
    int units[2] = {0, U - 1};
    float* Ku = (float*)malloc(sizeof(float) * 2 * (P ? P : 1) * d);
    float* Vu = (float*)malloc(sizeof(float) * 2 * (P ? P : 1) * d);
    synth_prefill_units(&w, 0, units, 2, Ku, Vu);
    CHECK(memcmp(Ku, Kp, sizeof(float) * (size_t)P * d) == 0);
    orc_kvm** ms = (orc_kvm**)malloc(sizeof(orc_kvm*) * U);
    for (int u = 0; u < U; ++u) {
        ms[u] = orc_new(G, d, ps, S, r, 0);
        CHECK(ms[u]);
        if (agg || rank_pinned) CHECK(orc_set_variant(ms[u], agg, rank_pinned) == 0);
        if (topk > 0) CHECK(orc_set_prompt_selection(ms[u], prompt_slots, topk) == 0);
        double* K = widen(Kp + (size_t)u * P * d, (size_t)P * d);
        double* V = widen(Vp + (size_t)u * P * d, (size_t)P * d);
        CHECK(orc_prefill(ms[u], P ? K : NULL, P ? V : NULL, P) == 0);
        free(K);
        free(V);
    }
    float* q = (float*)malloc(sizeof(float) * (size_t)T * U * G * d);
    float* k = (float*)malloc(sizeof(float) * (size_t)T * U * d);
    float* v = (float*)malloc(sizeof(float) * (size_t)T * U * d);
    synth_steps(&w, 0, 0, T, q, k, v);
    float* qu = (float*)malloc(sizeof(float) * (size_t)T * 2 * G * d);
    float* ku = (float*)malloc(sizeof(float) * (size_t)T * 2 * d);
    float* vu = (float*)malloc(sizeof(float) * (size_t)T * 2 * d);
    synth_steps_units(&w, 0, 0, T, units, 2, qu, ku, vu);
    CHECK(memcmp(qu, q, sizeof(float) * G * d) == 0);
    double* out = (double*)malloc(sizeof(double) * (size_t)U * G * d);
    int* pt = (int*)malloc(sizeof(int) * (size_t)U * S);
    int* ts = (int*)malloc(sizeof(int) * (size_t)U * S);
    int* st = (int*)malloc(sizeof(int) * S);
    int* fill = (int*)malloc(sizeof(int) * S);
    int* ev = (int*)malloc(sizeof(int) * U);
    int unit[6];
    double* sc = (double*)malloc(sizeof(double) * (size_t)U * S);
    double* th = (double*)malloc(sizeof(double) * U);
    double* pages = (double*)malloc(sizeof(double) * (size_t)S * ps * d * 2 + sizeof(double) * S * d * 2);
    int* att = (int*)malloc(sizeof(int) * S);
    for (int t = 0; t < T; ++t) {
        const float* qt = q + (size_t)t * U * G * d;
        const float* kt = k + (size_t)t * U * d;
        const float* vt = v + (size_t)t * U * d;
        if (grouped) {
            for (int b = 0; b < B; ++b) {
                double* qg = widen(qt + (size_t)b * H * G * d, (size_t)H * G * d);
                double* kg = widen(kt + (size_t)b * H * d, (size_t)H * d);
                double* vg = widen(vt + (size_t)b * H * d, (size_t)H * d);
                CHECK(orc_decode_group(ms + (size_t)b * H, H, qg, kg, vg, (t % 3) ? NULL : out) == 0);
                free(qg);
                free(kg);
                free(vg);
            }
        } else if (t % 5 == 4) { /* retention-only step with injected scores */
            double* inj = (double*)malloc(sizeof(double) * S);
            for (int u = 0; u < U; ++u) {
                for (int s = 0; s < S; ++s) inj[s] = (double)((s * 7 + t) % 5);
                CHECK(orc_decode(ms[u], NULL, NULL, NULL, NULL, inj) == 0);
            }
            free(inj);
        } else {
            CHECK(orc_decode_batch(ms, U, qt, kt, vt, (t % 2) ? NULL : out) == 0);
        }
        orc_state_batch(ms, U, pt, ts, ev);
        orc_scores_batch(ms, U, sc, th);
        for (int u = 0; u < U; ++u) {
            orc_state(ms[u], NULL, NULL, st, fill, unit);
            int resident = 0;
            for (int s = 0; s < S; ++s) resident += st[s] ? fill[s] : 0;
            CHECK(resident <= S * ps);
            /* adopting the oracle's own decision changes nothing */
            CHECK(orc_adopt_retention(ms[u], pt + (size_t)u * S, ts + (size_t)u * S, ev[u]) == 0);
            orc_last_attended(ms[u], att);
            orc_last_scores(ms[u], sc + (size_t)u * S, th + u);
        }
        if (t % 17 == 0) {
            double* Kx = pages;
            double* Vx = Kx + (size_t)S * ps * d;
            double* mn = Vx + (size_t)S * ps * d;
            orc_pages(ms[0], Kx, Vx, mn, mn + (size_t)S * d);
        }
    }
    int steps[64];
    CHECK(synth_active_milestones(&w, 0, 0, 0, T, steps, 64) >= 0);
    for (int u = 0; u < U; ++u) orc_free(ms[u]);
    free(ms);
    free(Kp), free(Vp), free(Ku), free(Vu), free(q), free(k), free(v), free(qu), free(ku), free(vu);
    free(out), free(pt), free(ts), free(st), free(fill), free(ev), free(sc), free(th), free(pages), free(att);
}

int main(void) {
    const uint32_t ctr[4] = {0, 0, 0, 0}, key[2] = {0, 0};
    uint32_t o[4];
    synth_philox4x32_10(ctr, key, o);
    CHECK(o[0] == 0x6627E8D5u);
    /* B H G d ps S P T r agg rank prompt_slots topk grouped outliers */
    run_case(2, 2, 4, 64, 16, 8, 40, 300, 0.5, 0, 0, 0, 0, 0, 0.0);       /* default rule */
    run_case(1, 2, 7, 128, 16, 16, 0, 200, 0.7, 0, 0, 0, 0, 0, 0.05);     /* no prompt, r 0.7, outliers */
    run_case(1, 1, 4, 64, 8, 300, 2300, 60, 0.5, 1, 1, 0, 0, 0, 0.0);     /* 300 slots, both variants */
    run_case(2, 1, 2, 32, 16, 6, 1000, 120, 0.25, 0, 0, 0, 0, 0, 0.0);    /* prompt over the budget */
    run_case(2, 2, 4, 64, 16, 14, 100, 200, 0.5, 0, 0, 8, 3, 0, 0.0);     /* Quest on the prompt */
    run_case(2, 4, 2, 64, 16, 8, 40, 150, 0.5, 1, 0, 0, 0, 1, 0.0);       /* one page table per sequence */
    run_case(1, 1, 16, 64, 128, 8, 300, 100, 1.0, 0, 1, 0, 0, 0, 0.0);    /* G 16, page 128, r 1 */
    printf("sanitized oracle and generator: ok\n");
    return 0;
}
