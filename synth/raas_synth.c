/*
 * Seeded synthetic inputs for the RaaS decode path (test and benchmark
 * infrastructure; holds none of the method's arithmetic).
 *
 * Every value is a pure function of (seed, layer, sequence, head, token,
 * element), so any (unit, step) can be regenerated on its own. The same
 * values feed the HIP path and the CPU oracle.
 *
 * Random bits: Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random
 * numbers: as easy as 1, 2, 3", SC 2011), written from its published
 * definition. Normals: Box-Muller on two 53-bit uniforms. Heavy-tailed key
 * outliers: Student-t with 3 degrees of freedom, t = z / sqrt(chi2_3 / 3).
 *
 * Structure (the paper's milestone pattern, Section 3.1 and Figure 3): a
 * milestone is an ordinary decode token whose key the queries of the next W
 * decode steps point towards. For those steps every query head of the unit
 * is q = |g| (0.8 u + 0.6 w), where g ~ N(0, I), u is the normalised sum of
 * the unit keys of all active milestones and w is the unit part of g
 * orthogonal to u; so cos(q, k_m) = 0.8 with one active milestone.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
    int32_t batch, n_layers, n_q_heads, n_kv_heads, head_dim;
    int32_t prefill_len;
    int32_t dtype;            /* 0: values rounded to fp32, 1: rounded to bf16 */
    int32_t ms_period;        /* milestone period R in decode steps; 0 = none */
    int32_t ms_phase_random;  /* 1: per-unit seeded phase in [0, R); 0: phase R-1 */
    int32_t ms_wmin, ms_wmax; /* window length ~ U{wmin..wmax} per milestone */
    double outlier_p;         /* per-key-element probability of a Student-t(3) draw */
    uint64_t seed;
} synth_workload;

enum {
    KIND_PREFILL_K = 1,
    KIND_PREFILL_V = 2,
    KIND_DECODE_Q = 3,
    KIND_DECODE_K = 4,
    KIND_DECODE_V = 5,
    KIND_MS_PHASE = 6,
    KIND_MS_WINDOW = 7,
    KIND_OUTLIER_PICK = 8,
    KIND_OUTLIER_T = 9,
};

/* ---- Philox4x32-10 ---- */
static inline void mulhilo32(uint32_t a, uint32_t b, uint32_t* hi, uint32_t* lo) {
    uint64_t p = (uint64_t)a * (uint64_t)b;
    *hi = (uint32_t)(p >> 32);
    *lo = (uint32_t)p;
}

static void philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4]) {
    uint32_t c0 = ctr_in[0], c1 = ctr_in[1], c2 = ctr_in[2], c3 = ctr_in[3];
    uint32_t k0 = key_in[0], k1 = key_in[1];
    for (int round = 0; round < 10; ++round) {
        uint32_t hi0, lo0, hi1, lo1;
        mulhilo32(0xD2511F53u, c0, &hi0, &lo0);
        mulhilo32(0xCD9E8D57u, c2, &hi1, &lo1);
        uint32_t n0 = hi1 ^ c1 ^ k0;
        uint32_t n1 = lo1;
        uint32_t n2 = hi0 ^ c3 ^ k1;
        uint32_t n3 = lo0;
        c0 = n0; c1 = n1; c2 = n2; c3 = n3;
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

static inline void draw(const synth_workload* w, uint32_t kind, uint32_t head, uint32_t layer,
                        uint32_t seq, uint32_t token, uint32_t idx, uint32_t out[4]) {
    uint32_t ctr[4] = {idx, token, (kind << 24) | (head & 0xFFFFFFu), (layer << 20) | (seq & 0xFFFFFu)};
    uint32_t key[2] = {(uint32_t)w->seed, (uint32_t)(w->seed >> 32)};
    philox4x32_10(ctr, key, out);
}

/* uniform in (0, 1) from two 32-bit words, 53 significant bits */
static inline double u53(uint32_t a, uint32_t b) {
    return ((double)(a >> 5) * 67108864.0 + (double)(b >> 6) + 0.5) * (1.0 / 9007199254740992.0);
}

/* two independent N(0,1) from one Philox block */
static inline void normal_pair(const uint32_t x[4], double* z0, double* z1) {
    double u1 = u53(x[0], x[1]);
    double u2 = u53(x[2], x[3]);
    double rad = sqrt(-2.0 * log(u1));
    double ang = 6.283185307179586476925286766559 * u2;
    *z0 = rad * cos(ang);
    *z1 = rad * sin(ang);
}

/* fills v[0..d) with N(0,1) draws of stream (kind, head, layer, seq, token) */
static void normal_vec(const synth_workload* w, uint32_t kind, uint32_t head, uint32_t layer,
                       uint32_t seq, uint32_t token, int d, double* v) {
    for (int e = 0; e < d; e += 2) {
        uint32_t x[4];
        draw(w, kind, head, layer, seq, token, (uint32_t)(e / 2), x);
        double z0, z1;
        normal_pair(x, &z0, &z1);
        v[e] = z0;
        if (e + 1 < d) v[e + 1] = z1;
    }
}

/* key vector: N(0,1), each element replaced by a Student-t(3) draw w.p. outlier_p */
static void key_vec(const synth_workload* w, uint32_t kind, uint32_t head, uint32_t layer,
                    uint32_t seq, uint32_t token, int d, double* v) {
    normal_vec(w, kind, head, layer, seq, token, d, v);
    if (w->outlier_p <= 0.0) return;
    uint32_t okind = KIND_OUTLIER_PICK, tkind = KIND_OUTLIER_T;
    /* distinct outlier streams for prefill and decode keys */
    uint32_t sub = (kind == KIND_PREFILL_K) ? 0u : 1u;
    for (int e = 0; e < d; ++e) {
        uint32_t x[4];
        draw(w, okind, head, layer, seq, token, ((uint32_t)e << 1) | sub, x);
        if (u53(x[0], x[1]) >= w->outlier_p) continue;
        uint32_t y[4], y2[4];
        draw(w, tkind, head, layer, seq, token, ((uint32_t)e << 2) | (sub << 1), y);
        draw(w, tkind, head, layer, seq, token, ((uint32_t)e << 2) | (sub << 1) | 1u, y2);
        double z, a, b, c;
        normal_pair(y, &z, &a);
        normal_pair(y2, &b, &c);
        double chi2 = a * a + b * b + c * c;
        v[e] = z / sqrt(chi2 / 3.0);
    }
}

static inline float round_to(int dtype, double x) {
    float f = (float)x; /* round to nearest even */
    if (dtype == 1) {
        uint32_t bits;
        memcpy(&bits, &f, 4);
        bits += 0x7FFFu + ((bits >> 16) & 1u);
        bits &= 0xFFFF0000u;
        memcpy(&f, &bits, 4);
    }
    return f;
}

/* prefill K, V of one unit (sequence b, KV head h): [prefill_len][head_dim] each */
static void unit_prefill(const synth_workload* w, int layer, int b, int h, float* K, float* V) {
    const int P = w->prefill_len, d = w->head_dim;
    double* tmp = (double*)malloc(sizeof(double) * (size_t)d);
    for (int t = 0; t < P; ++t) {
        size_t off = (size_t)t * d;
        key_vec(w, KIND_PREFILL_K, (uint32_t)h, (uint32_t)layer, (uint32_t)b, (uint32_t)t, d, tmp);
        for (int e = 0; e < d; ++e) K[off + e] = round_to(w->dtype, tmp[e]);
        normal_vec(w, KIND_PREFILL_V, (uint32_t)h, (uint32_t)layer, (uint32_t)b, (uint32_t)t, d, tmp);
        for (int e = 0; e < d; ++e) V[off + e] = round_to(w->dtype, tmp[e]);
    }
    free(tmp);
}

/* K, V: [batch][n_kv_heads][prefill_len][head_dim] */
void synth_prefill(const synth_workload* w, int layer, float* K, float* V) {
    const int B = w->batch, H = w->n_kv_heads;
    const size_t per = (size_t)w->prefill_len * w->head_dim;
#pragma omp parallel for collapse(2) schedule(static)
    for (int b = 0; b < B; ++b)
        for (int h = 0; h < H; ++h) unit_prefill(w, layer, b, h, K + ((size_t)b * H + h) * per, V + ((size_t)b * H + h) * per);
}

/* the same values for chosen units only (units[i] = sequence * n_kv_heads +
 * KV head): K, V [nu][prefill_len][head_dim] */
void synth_prefill_units(const synth_workload* w, int layer, const int* units, int nu, float* K, float* V) {
    const int H = w->n_kv_heads;
    const size_t per = (size_t)w->prefill_len * w->head_dim;
#pragma omp parallel for schedule(dynamic, 1)
    for (int i = 0; i < nu; ++i) unit_prefill(w, layer, units[i] / H, units[i] % H, K + (size_t)i * per, V + (size_t)i * per);
}

/* seeded phase of the unit's milestone schedule */
static int ms_phase(const synth_workload* w, int layer, int seq, int kvh) {
    if (!w->ms_phase_random) return w->ms_period - 1;
    uint32_t x[4];
    draw(w, KIND_MS_PHASE, (uint32_t)kvh, (uint32_t)layer, (uint32_t)seq, 0u, 0u, x);
    return (int)(x[0] % (uint32_t)w->ms_period);
}

static int ms_window(const synth_workload* w, int layer, int seq, int kvh, int index) {
    if (w->ms_wmax <= w->ms_wmin) return w->ms_wmin;
    uint32_t x[4];
    draw(w, KIND_MS_WINDOW, (uint32_t)kvh, (uint32_t)layer, (uint32_t)seq, (uint32_t)index, 0u, x);
    return w->ms_wmin + (int)(x[0] % (uint32_t)(w->ms_wmax - w->ms_wmin + 1));
}

/* number of milestones active at decode step t (m < t <= m + W_m); writes
 * their steps in increasing order when steps != NULL */
int synth_active_milestones(const synth_workload* w, int layer, int seq, int kvh, int t, int* steps,
                            int cap) {
    if (w->ms_period <= 0) return 0;
    const int R = w->ms_period, phase = ms_phase(w, layer, seq, kvh);
    int lo = t - w->ms_wmax;
    if (lo < 0) lo = 0;
    /* first milestone index i with phase + i*R >= lo */
    int i0 = (lo <= phase) ? 0 : (lo - phase + R - 1) / R;
    int n = 0;
    for (int i = i0;; ++i) {
        int m = phase + i * R;
        if (m >= t) break;
        if (t <= m + ms_window(w, layer, seq, kvh, i)) {
            if (steps && n < cap) steps[n] = m;
            ++n;
        }
    }
    return n;
}

/* decode inputs of one unit (sequence b, KV head h) at decode step t:
 * q [G][d] (the unit's query heads), k [d], v [d] */
static void unit_step(const synth_workload* w, int layer, int t, int b, int h, float* q, float* k, float* v) {
    const int d = w->head_dim, G = w->n_q_heads / w->n_kv_heads;
    const uint32_t tok = (uint32_t)t;
    double* tmp = (double*)malloc(sizeof(double) * (size_t)d * 3);
    double* u = tmp + d;
    double* mk = tmp + 2 * d;
    key_vec(w, KIND_DECODE_K, (uint32_t)h, (uint32_t)layer, (uint32_t)b, tok, d, tmp);
    for (int e = 0; e < d; ++e) k[e] = round_to(w->dtype, tmp[e]);
    normal_vec(w, KIND_DECODE_V, (uint32_t)h, (uint32_t)layer, (uint32_t)b, tok, d, tmp);
    for (int e = 0; e < d; ++e) v[e] = round_to(w->dtype, tmp[e]);

    /* direction u: normalised sum of the active milestones' unit keys */
    int steps[64];
    int na = synth_active_milestones(w, layer, b, h, t, steps, 64);
    if (na > 64) na = 64;
    for (int e = 0; e < d; ++e) u[e] = 0.0;
    for (int a = 0; a < na; ++a) {
        key_vec(w, KIND_DECODE_K, (uint32_t)h, (uint32_t)layer, (uint32_t)b, (uint32_t)steps[a], d, mk);
        double nn = 0.0;
        for (int e = 0; e < d; ++e) {
            mk[e] = (double)round_to(w->dtype, mk[e]);
            nn += mk[e] * mk[e];
        }
        nn = sqrt(nn);
        for (int e = 0; e < d; ++e) u[e] += mk[e] / nn;
    }
    double un = 0.0;
    for (int e = 0; e < d; ++e) un += u[e] * u[e];
    un = sqrt(un);
    for (int j = 0; j < G; ++j) {
        const int head = h * G + j;
        normal_vec(w, KIND_DECODE_Q, (uint32_t)head, (uint32_t)layer, (uint32_t)b, tok, d, tmp);
        if (na > 0 && un > 0.0) {
            double gn = 0.0, gu = 0.0;
            for (int e = 0; e < d; ++e) {
                gn += tmp[e] * tmp[e];
                gu += tmp[e] * (u[e] / un);
            }
            gn = sqrt(gn);
            double wn = 0.0;
            for (int e = 0; e < d; ++e) {
                double we = tmp[e] - gu * (u[e] / un);
                wn += we * we;
            }
            wn = sqrt(wn);
            for (int e = 0; e < d; ++e) {
                double we = (tmp[e] - gu * (u[e] / un)) / (wn > 0.0 ? wn : 1.0);
                tmp[e] = gn * (0.8 * (u[e] / un) + 0.6 * we);
            }
        }
        for (int e = 0; e < d; ++e) q[(size_t)j * d + e] = round_to(w->dtype, tmp[e]);
    }
    free(tmp);
}

/* q: [n][batch][n_q_heads][d]; k, v: [n][batch][n_kv_heads][d]; decode steps t0..t0+n-1 */
void synth_steps(const synth_workload* w, int layer, int t0, int n, float* q, float* k, float* v) {
    const int B = w->batch, H = w->n_kv_heads, d = w->head_dim;
    const int G = w->n_q_heads / H;
#pragma omp parallel for collapse(3) schedule(dynamic, 4)
    for (int s = 0; s < n; ++s)
        for (int b = 0; b < B; ++b)
            for (int h = 0; h < H; ++h) {
                const size_t uo = ((size_t)s * B + b) * H + h;
                unit_step(w, layer, t0 + s, b, h, q + uo * G * d, k + uo * d, v + uo * d);
            }
}

/* the same values for chosen units only: units[i] = sequence * n_kv_heads +
 * KV head; q: [n][nu][G][d]; k, v: [n][nu][d] */
void synth_steps_units(const synth_workload* w, int layer, int t0, int n, const int* units, int nu, float* q,
                       float* k, float* v) {
    const int H = w->n_kv_heads, d = w->head_dim;
    const int G = w->n_q_heads / H;
#pragma omp parallel for collapse(2) schedule(dynamic, 4)
    for (int s = 0; s < n; ++s)
        for (int i = 0; i < nu; ++i) {
            const size_t uo = (size_t)s * nu + i;
            unit_step(w, layer, t0 + s, units[i] / H, units[i] % H, q + uo * G * d, k + uo * d, v + uo * d);
        }
}

/* raw Philox block, exposed so tests can pin the generator to its published
 * known-answer vectors */
void synth_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
    philox4x32_10(ctr, key, out);
}
