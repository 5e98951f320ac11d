/*
 * Reference oracle for ResidualAttention over a disaggregated KV cache
 * (ForkKV, arXiv 2604.06370).
 *
 * TEST INFRASTRUCTURE ONLY.  The test suite, the smoke check and the
 * CPU-baseline leg of the benchmark are the only callers.  The product library
 * never loads this file and the two share no code, header, table or helper.
 *
 * What it computes (the plain definition, materialised, in fp64):
 *
 *   For every agent a and every logical key position p < L_a:
 *     K_a[p] = bCache_K[p] + RoPE_p( rCache_K,a[p] . B_K,a )          (1)
 *     V_a[p] = bCache_V[p] +         rCache_V,a[p] . B_V,a            (2)
 *   then, for every query row of agent a and every query head j (KV head
 *   h = j / (Hq/Hkv)), textbook softmax attention over the visible keys:
 *     s_p = scale * q_j . K_a[p]        for p <= position(query row)
 *     O_j = sum_p exp(s_p - max s) V_a[p] / sum_p exp(s_p - max s)      (3)
 *
 * Sources in the paper:
 *   (1),(2)  Section 2.2, Eq. 2: a projection is rebuilt as bCache + rCache x B_i,
 *            with bCache = xW and rCache = xA_i (Eq. 1, no extra scale factor).
 *   RoPE     Section 2.2 (last paragraph) and Section 5.1: RoPE is applied to the
 *            base key projection before it is cached, is not applied to the
 *            rCache, and is never applied to V (Fig. "Unified vs Disaggregated
 *            KV Cache" caption).  Section 5.3, "On-the-fly Key Reconstruction
 *            with Deferred RoPE": RoPE is applied to the up-projected LoRA key
 *            at the token's position, then added to the base key.
 *   (3)      Section 5.3: the fused kernel is stated to be exactly equal to plain
 *            attention over the reconstructed cache (Eq. 4, associativity), so the
 *            oracle is plain attention over the materialised K and V.
 *
 * Readings where the paper is silent (each is listed with its reason in the
 * design notes of the repository):
 *   - RoPE variant: rotate-half pairing (i, i + d/2), theta_i = base^(-2i/d),
 *     position = the key's logical index in its agent's sequence.
 *   - GQA: query head j reads KV head floor(j / (Hq/Hkv)).
 *   - rCache holds one r-vector per token for K and one for V, shared by all KV
 *     heads; B is r x (Hkv*d), and KV head h uses columns h*d .. h*d+d-1.
 *   - A query row at absolute position P sees keys 0..P (decode: P = L_a - 1).
 *
 * Layouts are logical (unpaged): the oracle never sees pages or block tables,
 * so page handling in the product is checked end to end against it.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

typedef struct {
    int32_t n_agents, hq, hkv, d, r;
    int32_t rope;             /* 1: rotate the LoRA part of K by RoPE (Section 5.3) */
    double rope_theta;        /* RoPE base */
    double scale;             /* softmax scale applied to q.k */
    const int64_t *seq_len;   /* [n_agents] L_a, keys held by agent a */
    const int64_t *key_offset;/* [n_agents] first entry of agent a in base_row / c_k / c_v */
    const int64_t *base_row;  /* [sum L_a] row of the base store holding agent a's key p */
    const double *base_k;     /* [n_rows][hkv][d] bCache keys (already RoPE'd) */
    const double *base_v;     /* [n_rows][hkv][d] bCache values */
    const double *c_k;        /* [sum L_a][r] rCache for K (x A_K) */
    const double *c_v;        /* [sum L_a][r] rCache for V (x A_V) */
    const double *b_k;        /* [n_agents][r][hkv*d] B_K of agent a's adapter */
    const double *b_v;        /* [n_agents][r][hkv*d] B_V of agent a's adapter */
    const int32_t *has_residual; /* [n_agents] 0: agent has no rCache (K = bCache) */
    const int64_t *q_offset;  /* [n_agents+1] query rows of agent a: q_offset[a] .. q_offset[a+1]-1 */
    const int64_t *q_pos;     /* [total_q] absolute position of each query row */
    const double *q;          /* [total_q][hq][d] queries (already RoPE'd) */
    double *out;              /* [total_q][hq][d] attention output */
} oracle_problem;

/* RoPE, rotate-half form: the pair (x[i], x[i+d/2]) is rotated by the angle
 * pos * theta_i with theta_i = base^(-2i/d).  The paper names no variant; this
 * is the reading used throughout (Section 5.3 applies "RoPE" to K_res.B_k). */
void oracle_rope_rotate(const double *x, int32_t d, int64_t pos, double base, double *out)
{
    int32_t half = d / 2;
    for (int32_t i = 0; i < half; ++i) {
        double theta = pow(base, -2.0 * (double)i / (double)d);
        double ang = (double)pos * theta;
        double c = cos(ang), s = sin(ang);
        double x0 = x[i], x1 = x[i + half];
        out[i] = x0 * c - x1 * s;
        out[i + half] = x1 * c + x0 * s;
    }
}

static int check_problem(const oracle_problem *p)
{
    if (p->n_agents < 0 || p->hq <= 0 || p->hkv <= 0 || p->d <= 0 || p->r < 0) return -1;
    if (p->hq % p->hkv != 0) return -2;
    if (p->rope && (p->d % 2) != 0) return -3;
    for (int32_t a = 0; a < p->n_agents; ++a) {
        if (p->seq_len[a] < 1) return -4;
        for (int64_t qi = p->q_offset[a]; qi < p->q_offset[a + 1]; ++qi)
            if (p->q_pos[qi] < 0 || p->q_pos[qi] >= p->seq_len[a]) return -5;
    }
    return 0;
}

/* Materialise K_a and V_a for one (agent, KV head) pair: equations (1), (2). */
static void build_kv(const oracle_problem *p, int32_t a, int32_t h, double *K, double *V,
                     double *u, double *ur)
{
    const int32_t d = p->d, r = p->r, n = p->hkv * p->d;
    const int64_t L = p->seq_len[a];
    const int64_t off = p->key_offset[a];
    const double *bk = p->b_k + (int64_t)a * r * n;
    const double *bv = p->b_v + (int64_t)a * r * n;
    for (int64_t t = 0; t < L; ++t) {
        const int64_t row = p->base_row[off + t];
        const double *kb = p->base_k + (row * p->hkv + h) * d;
        const double *vb = p->base_v + (row * p->hkv + h) * d;
        for (int32_t i = 0; i < d; ++i) { K[t * d + i] = kb[i]; V[t * d + i] = vb[i]; }
        if (!p->has_residual[a]) continue;
        const double *ck = p->c_k + (off + t) * r;
        const double *cv = p->c_v + (off + t) * r;
        /* u = rCache_K[t] . B_K restricted to head h's columns (Eq. 2) */
        for (int32_t i = 0; i < d; ++i) {
            double acc = 0.0;
            for (int32_t k = 0; k < r; ++k) acc += ck[k] * bk[(int64_t)k * n + h * d + i];
            u[i] = acc;
        }
        if (p->rope) {
            oracle_rope_rotate(u, d, t, p->rope_theta, ur);
            memcpy(u, ur, sizeof(double) * d);
        }
        for (int32_t i = 0; i < d; ++i) K[t * d + i] += u[i];
        /* value residual: rCache_V[t] . B_V, no RoPE */
        for (int32_t i = 0; i < d; ++i) {
            double acc = 0.0;
            for (int32_t k = 0; k < r; ++k) acc += cv[k] * bv[(int64_t)k * n + h * d + i];
            V[t * d + i] += acc;
        }
    }
}

/* Softmax attention of one query vector over keys 0..nvis-1: equation (3). */
static void attend(const double *qv, const double *K, const double *V, int64_t nvis, int32_t d,
                   double scale, double *s, double *o)
{
    double mx = -INFINITY;
    for (int64_t t = 0; t < nvis; ++t) {
        double acc = 0.0;
        for (int32_t i = 0; i < d; ++i) acc += qv[i] * K[t * d + i];
        s[t] = scale * acc;
        if (s[t] > mx) mx = s[t];
    }
    double z = 0.0;
    for (int64_t t = 0; t < nvis; ++t) { s[t] = exp(s[t] - mx); z += s[t]; }
    for (int32_t i = 0; i < d; ++i) o[i] = 0.0;
    for (int64_t t = 0; t < nvis; ++t)
        for (int32_t i = 0; i < d; ++i) o[i] += s[t] * V[t * d + i];
    for (int32_t i = 0; i < d; ++i) o[i] /= z;
}

/* Returns 0 on success, a negative code for an inconsistent problem, -100 when
 * memory runs out.  n_threads <= 0 uses the OpenMP default. */
int oracle_residual_attention(const oracle_problem *p, int32_t n_threads)
{
    int rc = check_problem(p);
    if (rc) return rc;
    const int32_t g = p->hq / p->hkv;
    const int64_t pairs = (int64_t)p->n_agents * p->hkv;
    int failed = 0;
#ifdef _OPENMP
    if (n_threads <= 0) n_threads = omp_get_max_threads();
#pragma omp parallel for schedule(dynamic, 1) num_threads(n_threads)
#endif
    for (int64_t ah = 0; ah < pairs; ++ah) {
        const int32_t a = (int32_t)(ah / p->hkv), h = (int32_t)(ah % p->hkv);
        const int64_t L = p->seq_len[a];
        const int32_t d = p->d;
        double *K = malloc(sizeof(double) * L * d);
        double *V = malloc(sizeof(double) * L * d);
        double *s = malloc(sizeof(double) * L);
        double *u = malloc(sizeof(double) * d);
        double *ur = malloc(sizeof(double) * d);
        if (!K || !V || !s || !u || !ur) {
#ifdef _OPENMP
#pragma omp atomic write
#endif
            failed = 1;
        } else {
            build_kv(p, a, h, K, V, u, ur);
            for (int64_t qi = p->q_offset[a]; qi < p->q_offset[a + 1]; ++qi) {
                const int64_t nvis = p->q_pos[qi] + 1;
                for (int32_t jj = 0; jj < g; ++jj) {
                    const int32_t j = h * g + jj;
                    attend(p->q + (qi * p->hq + j) * d, K, V, nvis, d, p->scale, s,
                           p->out + (qi * p->hq + j) * d);
                }
            }
        }
        free(K); free(V); free(s); free(u); free(ur);
    }
    return failed ? -100 : 0;
}

/* Number of threads the OpenMP runtime would use by default. */
int oracle_default_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
