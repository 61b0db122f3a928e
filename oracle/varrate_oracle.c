/*
 * VarRate CPU oracle (arXiv 2607.15498) -- TEST INFRASTRUCTURE.
 *
 * Only the tests, the smoke check and the bench's CPU-baseline leg may load or call this
 * library.  The product path (the HIP library under paper_2607_15498_amd/) never does, and
 * the two share no code.
 *
 * A plain, slow, obviously-correct fp64 implementation of the codec's data-parallel path,
 * written from the paper's definitions:
 *   attention              Sec. 3.1 "Preliminaries" (softmax of <q,k>/sqrt(d_h) over seen tokens)
 *   coded budget           Sec. 3.1 Eq. (3) "eq:budget"
 *   salience               Sec. 3.2 Eq. (4) "eq:salience" + length-5 moving average + min-max
 *   water-filling          Sec. 3.2 Eq. (5) "eq:waterfill", Algorithm 1 (REPEAT loop), footnote
 *                          on integer ranks
 *   projection/truncation  Sec. 3.3 Eq. (6) "eq:recon", Algorithm 1 (projection step)
 *   decode                 Sec. 4.4 "Cost": reconstruct-in-place, then stock attention
 *   coefficient quantiser  Sec. 3.3 "Composability": group-wise b-bit codes of the coefficients
 *   anchor residual codec  Sec. 3.1 "Residual codec" Eq. (2), Algorithm 1 (anchors, exact set,
 *                          nearest-anchor mean, residual)
 *
 * Specialisation (the data-parallel path only): per-KV-head bases P in R^{d x d} (R = d, so
 * full rank is exact), no anchors (residual mean zbar = 0), no RoPE, exact set = last w tokens.
 * Readings of points the paper leaves open are listed beside each function.
 *
 * Parity status: every function below is pinned by CPU tests against closed forms,
 * brute force, exact rational arithmetic or invariants (tests/test_oracle_*.py).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

#define EXPORT __attribute__((visibility("default")))

/* ------------------------------------------------------------------------------------- */
/* Eq. (3): B = D (kappa L - n_ref), with the per-head unit D -> d, L -> n, n_ref = w and
 * kappa given as an integer percent, floored to an integer number of coefficients.        */
EXPORT int64_t vro_budget(int64_t n, int64_t d, int64_t w, int64_t kappa_pct)
{
    int64_t full = kappa_pct * n * d;            /* kappa * L * D in units of 1/100 */
    int64_t kept = full >= 0 ? full / 100 : -((-full + 99) / 100);
    return kept - w * d;
}

EXPORT int vro_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Thread count of the OpenMP loops that follow (the timing harness's 1-thread baseline). */
EXPORT void vro_set_threads(int n)
{
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* ------------------------------------------------------------------------------------- */
/* Sec. 3.1 attention + Sec. 3.2 Eq. (4).
 * Window query i (0 <= i < w) sits at position p = n - w + i and attends causally to keys
 * 0..p.  Query head h reads KV head g = h / (H/G).  For every coded token t < N = n - w,
 *     s_t = (1 / (w H)) sum_i sum_h alpha_{i,h,t},
 *     alpha_{i,h,t} = exp(x_t - max_x) / sum_{t' <= p} exp(x_t' - max_x),
 *     x_t = <q_{i,h}, k_{t,g}> / sqrt(d).
 * Layouts: K [n][G][d], Qw [w][H][d] (row-major), s [N].                                 */
static double dot_fd(const float *a, const float *b, int d)
{
    double acc = 0.0;
    for (int c = 0; c < d; ++c) acc += (double)a[c] * (double)b[c];
    return acc;
}

EXPORT void vro_salience(int64_t n, int G, int H, int d, int w,
                         const float *K, const float *Qw, double *s)
{
    const int64_t N = n - w;
    const int rows = w * H;
    const int hpg = H / G;
    const double scale = 1.0 / sqrt((double)d);
    double *row_max = (double *)malloc(sizeof(double) * rows);
    double *row_sum = (double *)malloc(sizeof(double) * rows);

    /* pass 1: per (i, h) softmax normaliser over the causal range */
#pragma omp parallel for schedule(dynamic)
    for (int r = 0; r < rows; ++r) {
        const int i = r / H, h = r % H, g = h / hpg;
        const int64_t p = n - w + i;
        const float *q = Qw + ((int64_t)i * H + h) * d;
        double m = -INFINITY;
        for (int64_t t = 0; t <= p; ++t) {
            double x = dot_fd(q, K + (t * G + g) * d, d) * scale;
            if (x > m) m = x;
        }
        double z = 0.0;
        for (int64_t t = 0; t <= p; ++t)
            z += exp(dot_fd(q, K + (t * G + g) * d, d) * scale - m);
        row_max[r] = m;
        row_sum[r] = z;
    }
    /* pass 2: average of the normalised weights over the window and the heads */
    const double inv = 1.0 / ((double)w * (double)H);
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < N; ++t) {
        double acc = 0.0;
        for (int r = 0; r < rows; ++r) {
            const int i = r / H, h = r % H, g = h / hpg;
            const float *q = Qw + ((int64_t)i * H + h) * d;
            double x = dot_fd(q, K + (t * G + g) * d, d) * scale;
            acc += exp(x - row_max[r]) / row_sum[r];
        }
        s[t] = acc * inv;
    }
    free(row_max);
    free(row_sum);
}

/* ------------------------------------------------------------------------------------- */
/* Sec. 3.2: SnapKV's length-5 moving average over adjacent coded tokens (centred window,
 * terms outside [0, N) count as zero, always divided by 5), then rounded to fp32.  The fp32
 * array is the allocation input.                                                         */
EXPORT void vro_pool(const double *s, int64_t N, float *sbar)
{
    for (int64_t t = 0; t < N; ++t) {
        double acc = 0.0;
        for (int64_t k = t - 2; k <= t + 2; ++k)
            if (k >= 0 && k < N) acc += s[k];
        sbar[t] = (float)(acc / 5.0);
    }
}

/* Sec. 3.2: min-max normalisation over the coded set, s_hat in [0, 1], turned into exact
 * integer weights u_t = 1 + floor(s_hat * 2^24) in [1, 2^24 + 1].  Each fp64 operation is
 * rounded once (no contraction: this file is compiled with -ffp-contract=off).  A constant
 * signal (max == min, where min-max is 0/0) gives every token the same weight, which the
 * paper states collapses the allocation to the uniform-rank codec.                       */
EXPORT void vro_weights(const float *sbar, int64_t N, uint32_t *u)
{
    if (N <= 0) return;
    float mn = sbar[0], mx = sbar[0];
    for (int64_t t = 1; t < N; ++t) {
        if (sbar[t] < mn) mn = sbar[t];
        if (sbar[t] > mx) mx = sbar[t];
    }
    if (mx == mn) {
        for (int64_t t = 0; t < N; ++t) u[t] = (1u << 24) + 1u;
        return;
    }
    const double lo = (double)mn;
    const double range = (double)mx - lo;
    for (int64_t t = 0; t < N; ++t) {
        volatile double num = (double)sbar[t] - lo;
        volatile double shat = num / range;
        double scaled = shat * 16777216.0; /* exact: power of two */
        u[t] = 1u + (uint32_t)floor(scaled);
    }
}

/* ------------------------------------------------------------------------------------- */
/* Sec. 3.2 Eq. (5) + Algorithm 1 water-filling, solved in exact integer arithmetic.
 *   Continuous solution: q_t = clip(r_min + lambda u_t, r_min, R) with sum q_t = B.
 *   Sort u descending (ties: lower index first).  With the top k tokens capped at R,
 *   U(k) = the rest, Q(k) = sum_{U(k)} u, M(k) = B - R k - r_min (N - k); the uncapped
 *   tokens receive q_t = r_min + u_t M / Q.  Take the smallest k with
 *     (k == 0 or M u_(k) > (R - r_min) Q)  and  (k == N or (R - r_min) Q >= M u_(k+1)).
 *   This is the fixed point of Algorithm 1's clip-and-redistribute loop, which clips only
 *   tokens strictly above R.
 *   Integer ranks (footnote on integer ranks; reading: largest-remainder rounding so that
 *   sum r_t = B exactly): f_t = floor(q_t), remainder rho = B - sum f_t, and the rho uncapped
 *   tokens with the largest fractional parts phi_t = (u_t M) mod Q get +1; ties go to the
 *   larger u_t, then to the smaller index t.
 * Returns 0, or -2 when the budget is infeasible (N r_min > B or B > N R or N <= 0).
 * Optional outputs: the capped count k, M and Q.                                          */
typedef struct { uint32_t u; int64_t t; } ut_pair;

static int cmp_u_desc(const void *a, const void *b)
{
    const ut_pair *x = (const ut_pair *)a, *y = (const ut_pair *)b;
    if (x->u != y->u) return x->u > y->u ? -1 : 1;
    return x->t < y->t ? -1 : (x->t > y->t);
}

typedef struct { int64_t phi; uint32_t u; int64_t t; } frac_key;

static int cmp_frac_desc(const void *a, const void *b)
{
    const frac_key *x = (const frac_key *)a, *y = (const frac_key *)b;
    if (x->phi != y->phi) return x->phi > y->phi ? -1 : 1;
    if (x->u != y->u) return x->u > y->u ? -1 : 1;
    return x->t < y->t ? -1 : (x->t > y->t);
}

EXPORT int vro_allocate(const uint32_t *u, int64_t N, int64_t B, int r_min, int R,
                        int32_t *rank, int64_t *out_k, int64_t *out_M, int64_t *out_Q)
{
    if (N <= 0 || r_min < 0 || R < r_min) return -2;
    if ((__int128)N * r_min > B || (__int128)N * R < B) return -2;
    const int64_t D = (int64_t)R - r_min;

    ut_pair *ord = (ut_pair *)malloc(sizeof(ut_pair) * N);
    for (int64_t t = 0; t < N; ++t) { ord[t].u = u[t]; ord[t].t = t; }
    qsort(ord, N, sizeof(ut_pair), cmp_u_desc);

    /* suffix sums: tail[k] = sum of u over ord[k..N-1] = Q(k) */
    __int128 *tail = (__int128 *)malloc(sizeof(__int128) * (N + 1));
    tail[N] = 0;
    for (int64_t k = N - 1; k >= 0; --k) tail[k] = tail[k + 1] + ord[k].u;

    int64_t k = 0;
    __int128 M = 0, Q = 0;
    for (k = 0; k <= N; ++k) {
        Q = tail[k];
        M = (__int128)B - (__int128)R * k - (__int128)r_min * (N - k);
        int c1 = (k == 0) || (M * ord[k - 1].u > (__int128)D * Q);
        int c2 = (k == N) || ((__int128)D * Q >= M * ord[k].u);
        if (c1 && c2) break;
    }
    if (k > N) { free(ord); free(tail); return -2; } /* unreachable for feasible B */

    for (int64_t i = 0; i < k; ++i) rank[ord[i].t] = R;
    const int64_t nU = N - k;
    frac_key *fk = (frac_key *)malloc(sizeof(frac_key) * (nU > 0 ? nU : 1));
    __int128 sum_f = (__int128)R * k;
    for (int64_t i = 0; i < nU; ++i) {
        const ut_pair *p = &ord[k + i];
        __int128 num = (__int128)p->u * M;
        int64_t f = (int64_t)(num / Q);
        rank[p->t] = (int32_t)(r_min + f);
        sum_f += r_min + f;
        fk[i].phi = (int64_t)(num % Q);
        fk[i].u = p->u;
        fk[i].t = p->t;
    }
    int64_t rho = (int64_t)((__int128)B - sum_f);
    if (rho > 0) {
        qsort(fk, nU, sizeof(frac_key), cmp_frac_desc);
        for (int64_t i = 0; i < rho; ++i) rank[fk[i].t] += 1;
    }
    if (out_k) *out_k = k;
    if (out_M) *out_M = (int64_t)M;
    if (out_Q) *out_Q = (int64_t)Q;
    free(fk);
    free(ord);
    free(tail);
    return 0;
}

/* ------------------------------------------------------------------------------------- */
/* Storage rounding of a coefficient: nearest bfloat16 (8 significant bits), ties to even,
 * taken from the exact fp64 value; or nearest fp32.                                      */
static double round_bf16(double x)
{
    if (x == 0.0 || !isfinite(x)) return x;
    int e;
    double m = frexp(x, &e);              /* x = m 2^e, 0.5 <= |m| < 1 */
    double r = nearbyint(ldexp(m, 8));    /* 8 significant bits, ties-to-even */
    return ldexp(r, e - 8);
}

/* Sec. 3.3 Eq. (6), Algorithm 1 projection step: c_t = P x_t at full rank, then the nested
 * mask 1[j < r_t] keeps the leading r_t coefficients (0-based j).  Per KV head g:
 *     c[t][g][j] = sum_i P[g][j][i] X[t][g][i]   for j < rank[t], else 0,
 * rounded to the storage type (bf16 when storage_bf16 != 0, else fp32).
 * Layouts: X [n_tok][G][d], P [G][d][d] (row j = j-th direction), coef [n_tok][G][d].     */
EXPORT void vro_project(int64_t n_tok, int G, int d, const float *X, const float *P,
                        const int32_t *rank, int storage_bf16, float *coef)
{
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < n_tok; ++t) {
        for (int g = 0; g < G; ++g) {
            const float *x = X + (t * G + g) * d;
            float *c = coef + (t * G + g) * d;
            for (int j = 0; j < d; ++j) {
                if (j >= rank[t]) { c[j] = 0.0f; continue; }
                double acc = dot_fd(P + ((int64_t)g * d + j) * d, x, d);
                c[j] = storage_bf16 ? (float)round_bf16(acc) : (float)acc;
            }
        }
    }
}

/* ------------------------------------------------------------------------------------- */
/* Sec. 3.1 "Joint per-token vector" and Algorithm 1 (first and last steps): rotary position
 * embedding in the rotate-half layout.  Coordinates i and i + d/2 form pair i; at position p
 * the pair turns by the angle sign * p * theta[i] (exact product, fp64):
 *     y_i       = x_i cos(a) - x_{i+d/2} sin(a)
 *     y_{i+d/2} = x_i sin(a) + x_{i+d/2} cos(a).
 * sign = +1 applies the embedding (pre-RoPE -> post-RoPE), sign = -1 removes it.
 * Layouts: X, out [n_tok][G][d]; pos [n_tok]; theta [d/2].                                */
static void rope_row(const double *x, double *y, int d, double p, const float *theta, int sign)
{
    const int h = d / 2;
    for (int i = 0; i < h; ++i) {
        const double a = (double)sign * p * (double)theta[i];
        const double c = cos(a), s = sin(a);
        const double x0 = x[i], x1 = x[i + h];
        y[i] = x0 * c - x1 * s;
        y[i + h] = x0 * s + x1 * c;
    }
}

EXPORT void vro_rope(int64_t n_tok, int G, int d, const float *X, const int64_t *pos,
                     const float *theta, int sign, double *out)
{
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < n_tok; ++t) {
        double x[512];
        for (int g = 0; g < G; ++g) {
            for (int i = 0; i < d; ++i) x[i] = (double)X[(t * G + g) * d + i];
            rope_row(x, out + (t * G + g) * d, d, (double)pos[t], theta, sign);
        }
    }
}

/* Sec. 4.4 decode, reconstruct-in-place: coded tokens are rebuilt from their stored
 * coefficients, x_hat_t = P^T (m_t . c_t) (Eq. 6 with zbar = 0); exact tokens (the window
 * and any tokens appended during decode) are used as stored.  A decode query then runs
 * stock attention over all of them:
 *     o_h = sum_t softmax_t(<q_h, k_hat_t> / sqrt(d)) v_hat_t        (fp64).
 * With rotary embedding (pos != NULL; the last step of Algorithm 1), a coded key is
 * re-rotated to post-RoPE at its token position pos[t] after the reconstruction; the exact
 * rows and the query are post-RoPE already.
 * Layouts: coefK/coefV [N][G][d] (zero beyond the rank), Kx/Vx [n_exact][G][d],
 * PK/PV [G][d][d], q [H][d], out [H][d].                                                  */
static void decode_impl(int64_t N, int64_t n_exact, int G, int H, int d,
                        const float *coefK, const float *coefV, const int32_t *rank,
                        const float *Kx, const float *Vx, const float *PK, const float *PV,
                        const float *q, const int64_t *pos, const float *theta, double *out)
{
    const int hpg = H / G;
    const double scale = 1.0 / sqrt((double)d);
    const int64_t T = N + n_exact;
    double *kh = (double *)malloc(sizeof(double) * (size_t)(N > 0 ? N : 1) * d);
    double *vh = (double *)malloc(sizeof(double) * (size_t)(N > 0 ? N : 1) * d);
    double *x = (double *)malloc(sizeof(double) * (size_t)(T > 0 ? T : 1));

    for (int g = 0; g < G; ++g) {
        const float *Pk = PK + (int64_t)g * d * d;
        const float *Pv = PV + (int64_t)g * d * d;
#pragma omp parallel for schedule(static)
        for (int64_t t = 0; t < N; ++t) {
            const float *ck = coefK + (t * G + g) * d;
            const float *cv = coefV + (t * G + g) * d;
            double kt[512];
            for (int c = 0; c < d; ++c) {
                double ak = 0.0, av = 0.0;
                for (int j = 0; j < rank[t]; ++j) {
                    ak += (double)ck[j] * (double)Pk[(int64_t)j * d + c];
                    av += (double)cv[j] * (double)Pv[(int64_t)j * d + c];
                }
                kt[c] = ak;
                vh[t * d + c] = av;
            }
            if (pos) rope_row(kt, kh + t * d, d, (double)pos[t], theta, +1);
            else for (int c = 0; c < d; ++c) kh[t * d + c] = kt[c];
        }
        for (int hh = 0; hh < hpg; ++hh) {
            const int h = g * hpg + hh;
            const float *qh = q + (int64_t)h * d;
            double m = -INFINITY;
            for (int64_t t = 0; t < T; ++t) {
                double acc = 0.0;
                if (t < N) {
                    for (int c = 0; c < d; ++c) acc += (double)qh[c] * kh[t * d + c];
                } else {
                    acc = dot_fd(qh, Kx + ((t - N) * G + g) * d, d);
                }
                x[t] = acc * scale;
                if (x[t] > m) m = x[t];
            }
            double z = 0.0;
            for (int64_t t = 0; t < T; ++t) { x[t] = exp(x[t] - m); z += x[t]; }
            double *o = out + (int64_t)h * d;
            for (int c = 0; c < d; ++c) o[c] = 0.0;
            for (int64_t t = 0; t < T; ++t) {
                const double a = x[t] / z;
                if (t < N) {
                    for (int c = 0; c < d; ++c) o[c] += a * vh[t * d + c];
                } else {
                    const float *v = Vx + ((t - N) * G + g) * d;
                    for (int c = 0; c < d; ++c) o[c] += a * (double)v[c];
                }
            }
        }
    }
    free(kh);
    free(vh);
    free(x);
}

EXPORT void vro_decode(int64_t N, int64_t n_exact, int G, int H, int d,
                       const float *coefK, const float *coefV, const int32_t *rank,
                       const float *Kx, const float *Vx, const float *PK, const float *PV,
                       const float *q, double *out)
{
    decode_impl(N, n_exact, G, H, d, coefK, coefV, rank, Kx, Vx, PK, PV, q, NULL, NULL, out);
}

EXPORT void vro_decode_rope(int64_t N, int64_t n_exact, int G, int H, int d,
                            const float *coefK, const float *coefV, const int32_t *rank,
                            const float *Kx, const float *Vx, const float *PK, const float *PV,
                            const float *q, const int64_t *pos, const float *theta, double *out)
{
    decode_impl(N, n_exact, G, H, d, coefK, coefV, rank, Kx, Vx, PK, PV, q, pos, theta, out);
}

/* ------------------------------------------------------------------------------------- */
/* Sec. 3.3 "Composability": the coefficients are themselves quantised, group-wise, to b
 * bits, with the allocation unchanged.  Reading (the paper names only "standard group-wise
 * b-bit quantization"): symmetric absmax groups; a group is one token's coefficients of one
 * head and one stream (K or V) in one 32-coordinate segment [32 s, min(32 s + 32, r_t)).
 * With Qmax = 2^(b-1) - 1 the group's scale is
 *     sc = half(fp32(amax / Qmax))          (IEEE fp32 division, then nearest binary16)
 * and each coefficient x of the group gets the code
 *     k = clamp(rint(fp32(x / sc)), -Qmax, Qmax)    (IEEE fp32 division, ties to even),
 * read back as k * sc.  A group whose scale is 0 codes every entry as 0; entries past the
 * token's rank are 0.  The input x is the stored (storage-rounded) coefficient.            */

/* Nearest IEEE 754 binary16 value (ties to even) of an fp32 value, returned as fp32:
 * 11 significant bits for |x| >= 2^-14, a fixed quantum of 2^-24 below that (subnormals),
 * infinity past the largest finite value 65504.                                          */
EXPORT float vro_half_round(float x)
{
    if (x == 0.0f || !isfinite(x)) return x;
    int e;
    (void)frexp((double)x, &e);             /* |x| = m 2^e, 0.5 <= m < 1 */
    int qexp = e - 11;                      /* quantum of an 11-bit significand */
    if (qexp < -24) qexp = -24;             /* subnormal range */
    double r = nearbyint(ldexp((double)x, -qexp)) ;
    double y = ldexp(r, qexp);
    if (fabs(y) > 65504.0) return x > 0 ? INFINITY : -INFINITY;
    return (float)y;
}

EXPORT void vro_quantize(int64_t n_tok, int G, int d, const float *coef, const int32_t *rank,
                         int bits, int8_t *codes, float *scales, float *deq)
{
    const int qmax = (1 << (bits - 1)) - 1;
    const int nseg = (d + 31) / 32;
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < n_tok; ++t) {
        for (int g = 0; g < G; ++g) {
            const float *x = coef + (t * G + g) * d;
            int8_t *k = codes + (t * G + g) * d;
            float *y = deq + (t * G + g) * d;
            for (int j = 0; j < d; ++j) { k[j] = 0; y[j] = 0.0f; }
            for (int sg = 0; sg < nseg; ++sg) {
                const int lo = 32 * sg;
                int hi = lo + 32 < rank[t] ? lo + 32 : rank[t];
                if (hi > d) hi = d;
                float amax = 0.0f;
                for (int j = lo; j < hi; ++j) {
                    const float a = fabsf(x[j]);
                    if (a > amax) amax = a;
                }
                volatile float ratio = amax / (float)qmax;
                const float sc = vro_half_round(ratio);
                scales[(t * G + g) * nseg + sg] = sc;
                if (sc == 0.0f) continue;
                for (int j = lo; j < hi; ++j) {
                    volatile float q = x[j] / sc;
                    float r = nearbyintf(q);
                    if (r > (float)qmax) r = (float)qmax;
                    if (r < -(float)qmax) r = -(float)qmax;
                    k[j] = (int8_t)r;
                    y[j] = r * sc;
                }
            }
        }
    }
}

/* ------------------------------------------------------------------------------------- */
/* Sec. 3.1 "Residual codec" (Eq. 2) and Algorithm 1 (anchors, exact set, residual).
 * Anchors: the prefix tokens at stride delta, t = 0, delta, 2 delta, ... < N (the paper's
 * z_1, z_{1+delta}, ... in 1-based numbering); they are kept exact, as is the window.
 * Joint vector z_t = [k_t (all G heads); v_t (all G heads)] in R^{2 G d}.  For every other
 * prefix token, its c nearest anchors in Euclidean distance over z (computed exactly in fp64
 * here; ties to the lower anchor number).  anchor_of[t] = index of t in the anchor list, or
 * -1; nn[t][0..c-1] = anchor numbers in increasing distance (rows of anchors left -1).     */
EXPORT void vro_anchor_nearest(int64_t N, int G, int d, int delta, int c, const float *K, const float *V,
                               int32_t *nn, double *dist)
{
    const int64_t na = (N + delta - 1) / delta;
    const int64_t D = (int64_t)G * d;
#pragma omp parallel for schedule(dynamic, 64)
    for (int64_t t = 0; t < N; ++t) {
        int32_t *out = nn + t * c;
        double *od = dist + t * c;
        for (int k = 0; k < c; ++k) { out[k] = -1; od[k] = INFINITY; }
        if (t % delta == 0) continue;
        for (int64_t a = 0; a < na; ++a) {
            const int64_t ta = a * delta;
            double s = 0.0;
            for (int64_t i = 0; i < D; ++i) {
                const double dk = (double)K[t * D + i] - (double)K[ta * D + i];
                const double dv = (double)V[t * D + i] - (double)V[ta * D + i];
                s += dk * dk + dv * dv;
            }
            /* insert into the sorted list (strictly smaller moves ahead: ties keep the
             * lower anchor number, which was seen first) */
            int pos = c;
            while (pos > 0 && s < od[pos - 1]) --pos;
            if (pos < c) {
                for (int k = c - 1; k > pos; --k) { od[k] = od[k - 1]; out[k] = out[k - 1]; }
                od[pos] = s;
                out[pos] = (int32_t)a;
            }
        }
    }
}

/* Decode with anchors (reconstruct-in-place, Eq. 6 with the anchor mean):
 *   coded token i (token index tok[i]): k_hat = (1/c) sum_k Ka[nn[i][k]] + P_K^T (m . cK[i]),
 *                                       v_hat likewise;
 *   anchors (Ka, Va) and exact rows (Kx, Vx) as stored;
 * then stock attention of q over all of them (fp64).  Layouts: coefK/coefV [Nc][G][d],
 * nn [Nc][c] anchor numbers, Ka/Va [na][G][d], Kx/Vx [n_exact][G][d], q [H][d], out [H][d]. */
EXPORT void vro_decode_anchor(int64_t Nc, int64_t na, int64_t n_exact, int G, int H, int d, int c,
                              const float *coefK, const float *coefV, const int32_t *rank,
                              const int32_t *nn, const float *Ka, const float *Va,
                              const float *Kx, const float *Vx, const float *PK, const float *PV,
                              const float *q, double *out)
{
    const int hpg = H / G;
    const double scale = 1.0 / sqrt((double)d);
    const int64_t T = Nc + na + n_exact;
    double *kh = (double *)malloc(sizeof(double) * (size_t)(Nc > 0 ? Nc : 1) * d);
    double *vh = (double *)malloc(sizeof(double) * (size_t)(Nc > 0 ? Nc : 1) * d);
    double *x = (double *)malloc(sizeof(double) * (size_t)(T > 0 ? T : 1));
    for (int g = 0; g < G; ++g) {
        const float *Pk = PK + (int64_t)g * d * d;
        const float *Pv = PV + (int64_t)g * d * d;
#pragma omp parallel for schedule(static)
        for (int64_t i = 0; i < Nc; ++i) {
            const float *ck = coefK + (i * G + g) * d;
            const float *cv = coefV + (i * G + g) * d;
            for (int e = 0; e < d; ++e) {
                double mk = 0.0, mv = 0.0;
                for (int k = 0; k < c; ++k) {
                    const int64_t a = nn[i * c + k];
                    mk += (double)Ka[(a * G + g) * d + e];
                    mv += (double)Va[(a * G + g) * d + e];
                }
                double ak = mk / c, av = mv / c;
                for (int j = 0; j < rank[i]; ++j) {
                    ak += (double)ck[j] * (double)Pk[(int64_t)j * d + e];
                    av += (double)cv[j] * (double)Pv[(int64_t)j * d + e];
                }
                kh[i * d + e] = ak;
                vh[i * d + e] = av;
            }
        }
        for (int hh = 0; hh < hpg; ++hh) {
            const int h = g * hpg + hh;
            const float *qh = q + (int64_t)h * d;
            double m = -INFINITY;
            for (int64_t t = 0; t < T; ++t) {
                double acc = 0.0;
                if (t < Nc) {
                    for (int e = 0; e < d; ++e) acc += (double)qh[e] * kh[t * d + e];
                } else if (t < Nc + na) {
                    acc = dot_fd(qh, Ka + ((t - Nc) * G + g) * d, d);
                } else {
                    acc = dot_fd(qh, Kx + ((t - Nc - na) * G + g) * d, d);
                }
                x[t] = acc * scale;
                if (x[t] > m) m = x[t];
            }
            double z = 0.0;
            for (int64_t t = 0; t < T; ++t) { x[t] = exp(x[t] - m); z += x[t]; }
            double *o = out + (int64_t)h * d;
            for (int e = 0; e < d; ++e) o[e] = 0.0;
            for (int64_t t = 0; t < T; ++t) {
                const double a = x[t] / z;
                if (t < Nc) {
                    for (int e = 0; e < d; ++e) o[e] += a * vh[t * d + e];
                } else {
                    const float *v = t < Nc + na ? Va + ((t - Nc) * G + g) * d : Vx + ((t - Nc - na) * G + g) * d;
                    for (int e = 0; e < d; ++e) o[e] += a * (double)v[e];
                }
            }
        }
    }
    free(kh);
    free(vh);
    free(x);
}

/* ------------------------------------------------------------------------------------- */
/* Sec. 3.1 Eq. (1) "Joint per-token vector" with one shared basis: z_t = [k_t of all G heads;
 * v_t of all G heads] in R^Dz, Dz = 2 G d, and a basis W in R^{R x Dz} (row j = j-th
 * direction).  Eq. (6): c_t = W z_t at full rank, the leading rank[t] coefficients kept, the
 * rest 0, rounded to the storage type.  Layouts: K, V [n_tok][G][d]; W [R][Dz];
 * coef [n_tok][R].                                                                         */
EXPORT void vro_project_joint(int64_t n_tok, int G, int d, int R, const float *K, const float *V,
                              const float *W, const int32_t *rank, int storage_bf16, float *coef)
{
    const int half = G * d, Dz = 2 * G * d;
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < n_tok; ++t) {
        const float *kt = K + t * half, *vt = V + t * half;
        float *c = coef + t * R;
        for (int j = 0; j < R; ++j) {
            if (j >= rank[t]) { c[j] = 0.0f; continue; }
            const float *w = W + (int64_t)j * Dz;
            double acc = dot_fd(w, kt, half) + dot_fd(w + half, vt, half);
            c[j] = storage_bf16 ? (float)round_bf16(acc) : (float)acc;
        }
    }
}

/* Sec. 4.4 decode, reconstruct-in-place, shared basis: z_hat_t = W^T (m_t . c_t) split into
 * the keys and values of every head (Eq. 6 with zbar = 0); exact rows as stored; then stock
 * attention per query head h over KV head h / (H / G), fp64.
 * Layouts: coef [N][R], Kx/Vx [n_exact][G][d], W [R][Dz], q [H][d], out [H][d].            */
EXPORT void vro_decode_joint(int64_t N, int64_t n_exact, int G, int H, int d, int R,
                             const float *coef, const int32_t *rank, const float *Kx, const float *Vx,
                             const float *W, const float *q, double *out)
{
    const int hpg = H / G, half = G * d, Dz = 2 * G * d;
    const double scale = 1.0 / sqrt((double)d);
    const int64_t T = N + n_exact;
    double *zh = (double *)malloc(sizeof(double) * (size_t)(N > 0 ? N : 1) * Dz);
    double *x = (double *)malloc(sizeof(double) * (size_t)(T > 0 ? T : 1));
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < N; ++t) {
        const float *c = coef + t * R;
        double *z = zh + t * Dz;
        for (int i = 0; i < Dz; ++i) z[i] = 0.0;
        for (int j = 0; j < rank[t]; ++j) {
            const float *w = W + (int64_t)j * Dz;
            for (int i = 0; i < Dz; ++i) z[i] += (double)c[j] * (double)w[i];
        }
    }
    for (int h = 0; h < H; ++h) {
        const int g = h / hpg;
        const float *qh = q + (int64_t)h * d;
        double m = -INFINITY;
        for (int64_t t = 0; t < T; ++t) {
            double acc = 0.0;
            if (t < N) {
                const double *k = zh + t * Dz + (int64_t)g * d;
                for (int i = 0; i < d; ++i) acc += (double)qh[i] * k[i];
            } else {
                acc = dot_fd(qh, Kx + ((t - N) * G + g) * d, d);
            }
            x[t] = acc * scale;
            if (x[t] > m) m = x[t];
        }
        double zs = 0.0;
        for (int64_t t = 0; t < T; ++t) { x[t] = exp(x[t] - m); zs += x[t]; }
        double *o = out + (int64_t)h * d;
        for (int i = 0; i < d; ++i) o[i] = 0.0;
        for (int64_t t = 0; t < T; ++t) {
            const double a = x[t] / zs;
            if (t < N) {
                const double *v = zh + t * Dz + half + (int64_t)g * d;
                for (int i = 0; i < d; ++i) o[i] += a * v[i];
            } else {
                const float *v = Vx + ((t - N) * G + g) * d;
                for (int i = 0; i < d; ++i) o[i] += a * (double)v[i];
            }
        }
    }
    free(zh);
    free(x);
}
