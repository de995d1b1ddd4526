/*
 * vkvref.c -- fp64 CPU oracle for the VestigeKV decode-time hot path.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may link, load or
 * call this file: only tests/, the smoke entry point and the bench's
 * cpu_baseline leg use it.  It shares no code, header, table or helper with
 * the HIP library; the two meet only through seeded inputs.
 *
 * What it computes (VestigeKV, arXiv 2609.03949):
 *   - cache row  C_u = [c_u (512 latent) ; r_u (64 branch)]           Sec. 3, Eq. (setup)
 *   - index row  (r_u, P c_u, eta_u) with a rank-r basis P             Sec. 4.2 (index entry)
 *   - index score  q_r.r_u + (P q_c).(P c_u), the first two terms of    Sec. 4.2, Eq. (trigger)
 *     the trigger, maximised over heads; top-k by (score desc, index asc)
 *   - Cauchy-Schwarz certificate of the sketch residual                 Lemma (Index certificate)
 *   - exact softmax attention over the attended multiset                Lemma (Exchangeability)
 *   - per-page boxes of index rows and the interval bound of a page     App. (dividend inside prior
 *                                                                        algorithms), page-bound pruning
 *
 * Every floating-point step is fp64 with an explicitly stated order (a
 * plain sequential dot product), so that it is a fixed function of the
 * bf16 input bits.  Readings where the paper is silent are stated beside
 * the function that takes them.  Compile with -ffp-contract=off.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define D_LAT 512
#define D_ROPE 64
#define D_ROW 576

/* Margin used to turn fp64 norm computations into rigorous upper bounds:
 * 2^-40 is more than 16x the worst-case relative error of a 512-term fp64
 * dot product (512 * 2^-53 = 2^-44). */
#define VKVREF_G 0x1p-40

/* ---------------------------------------------------------------- bf16 */

double vkvref_bf16_to_f64(uint16_t b) {
    uint32_t u = ((uint32_t)b) << 16;
    float f;
    memcpy(&f, &u, 4);
    return (double)f;
}

/* Round an fp64 value to bf16, round-to-nearest-even, in ONE rounding
 * (no detour through fp32, which would round twice). */
uint16_t vkvref_round_bf16(double x) {
    if (x != x) return 0x7FC0;
    uint16_t sign = signbit(x) ? 0x8000 : 0;
    double ax = fabs(x);
    if (ax == 0.0) return sign;
    /* halfway between the largest finite bf16 (2-2^-7)*2^127 and 2^128 */
    if (ax >= ldexp(2.0 - ldexp(1.0, -8), 127)) return (uint16_t)(sign | 0x7F80);
    int e;
    frexp(ax, &e);               /* ax in [2^(e-1), 2^e) */
    int E = e - 1;
    int qexp = (E >= -126) ? (E - 7) : -133;   /* quantum of the bf16 grid at ax */
    double q = ldexp(ax, -qexp);               /* exact: power-of-two scaling */
    double fl = floor(q);
    double frac = q - fl;                      /* exact */
    double rn;
    if (frac > 0.5) rn = fl + 1.0;
    else if (frac < 0.5) rn = fl;
    else rn = (fmod(fl, 2.0) == 0.0) ? fl : fl + 1.0;
    double res = ldexp(rn, qexp);              /* exactly representable in bf16 */
    float f = (float)res;
    uint32_t u;
    memcpy(&u, &f, 4);
    return (uint16_t)(sign | (u >> 16));
}

/* Smallest float f with (double)f >= x (rounding toward +infinity). */
float vkvref_ru_f32(double x) {
    float f = (float)x;
    if ((double)f < x) f = nextafterf(f, INFINITY);
    return f;
}

/* Smallest float f >= 0 with f*f >= x, evaluated exactly: the square of a
 * float is exact in fp64, so the result does not depend on how sqrt rounds. */
float vkvref_ru_sqrt_f32(double x) {
    if (!(x > 0.0)) return 0.0f;
    float f = (float)sqrt(x);
    while ((double)f * (double)f < x) f = nextafterf(f, INFINITY);
    for (;;) {
        float p = nextafterf(f, 0.0f);
        if ((double)p * (double)p >= x) f = p;
        else break;
    }
    return f;
}

/* ------------------------------------------------------- digest basis P */

/* Gershgorin certificate that the bf16 basis is contractive (||P||_2 <= 1),
 * which makes M = I - P^T P positive semidefinite so that Cauchy-Schwarz in
 * the M-seminorm bounds the sketch residual (Lemma (Index certificate)).
 * Returns the Gershgorin bound max_j sum_k |(P P^T)_jk| computed in fp64. */
double vkvref_gershgorin(const uint16_t* P, int r) {
    double best = 0.0;
    for (int j = 0; j < r; ++j) {
        double row = 0.0;
        for (int k = 0; k < r; ++k) {
            double g = 0.0;
            for (int i = 0; i < D_LAT; ++i)
                g = fma(vkvref_bf16_to_f64(P[(int64_t)j * D_LAT + i]),
                        vkvref_bf16_to_f64(P[(int64_t)k * D_LAT + i]), g);
            row += fabs(g);
        }
        if (row > best) best = row;
    }
    return best;
}

/* ------------------------------------------------- projection + scalars */

/* Project one 512-vector v with P: w_j = sum_i P[j,i] v[i] (fp64, i
 * ascending), digest d_j = RNE_bf16(w_j).  Then the three certificate
 * scalars, each rounded up to fp32 (Lemma (Index certificate), with the
 * bf16 rounding of the stored sketch accounted for):
 *   resid >= sqrt(v^T (I - P^T P) v)   (eta_u for a row, a_h for a head)
 *   dnorm >= ||d||                      (used for heads: ||qd_h||)
 *   derr  >= ||d - P v||                (eps_u for a row, e_h for a head)
 *   pnorm >= ||P v||                    (gamma_u for a row)
 * The fp64 values carry rounding error; the margins G make them upper
 * bounds of the exact real quantities.  The bound on ||P v - w|| uses
 * ||P||_F^2 <= r, which holds for every contractive basis (the only case in
 * which the scalars are used). */
static void project_and_bound(const double* v, const uint16_t* P, int r, uint16_t* d, float* resid, float* dnorm, float* derr,
                              float* pnorm) {
    double w[D_LAT];
    double Nv = 0.0;
    for (int i = 0; i < D_LAT; ++i) Nv = fma(v[i], v[i], Nv);
    for (int j = 0; j < r; ++j) {
        double acc = 0.0;
        for (int i = 0; i < D_LAT; ++i)
            acc = fma(vkvref_bf16_to_f64(P[(int64_t)j * D_LAT + i]), v[i], acc);
        w[j] = acc;
        d[j] = vkvref_round_bf16(acc);
    }
    double Nw = 0.0, Ne = 0.0, Nd = 0.0;
    for (int j = 0; j < r; ++j) Nw = fma(w[j], w[j], Nw);
    for (int j = 0; j < r; ++j) {
        double t = vkvref_bf16_to_f64(d[j]) - w[j];
        Ne = fma(t, t, Ne);
    }
    for (int j = 0; j < r; ++j) {
        double dj = vkvref_bf16_to_f64(d[j]);
        Nd = fma(dj, dj, Nd);
    }
    const double G = VKVREF_G;
    double Dm = G * (double)vkvref_ru_sqrt_f32((double)r * Nv);   /* >= ||P v - w|| */
    double sw = (double)vkvref_ru_sqrt_f32(Nw);
    double X = ((Nv - Nw) + G * (Nv + Nw)) + (2.0 * Dm) * sw;
    *resid = vkvref_ru_sqrt_f32((X > 0.0 ? X : 0.0) * (1.0 + G));
    *pnorm = vkvref_ru_f32(sw * (1.0 + G) + Dm);
    *derr = vkvref_ru_f32((double)vkvref_ru_sqrt_f32(Ne) * (1.0 + G) + Dm);
    *dnorm = vkvref_ru_sqrt_f32(Nd * (1.0 + G));
}

/* Index build (the compression event's tier-2 index, Sec. 4.2 and the
 * appendix's request lifecycle): for every row u of every sequence,
 *   index[b,u,:] = [ r_u (bit copy, if with_rope) ; RNE_bf16(P c_u) ]
 * and, if eta is non-null, the row certificate scalars eta_u, eps_u, gamma_u.
 * Reading: the paper draws P from the context's own queries; here P is an
 * input.  r may be 0 (no sketch: eta_u >= ||c_u||, eps_u = gamma_u = 0). */
int vkvref_digest_build(const uint16_t* cache, int64_t B, int64_t T, int64_t row_stride,
                        const uint16_t* P, int r, int with_rope, uint16_t* index,
                        int64_t index_stride, float* eta, float* eps, float* gam,
                        int nthreads) {
    int64_t n = (int64_t)B * T;
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(static)
#endif
    for (int64_t ru = 0; ru < n; ++ru) {
        const uint16_t* row = cache + ru * row_stride;
        double c[D_LAT];
        for (int i = 0; i < D_LAT; ++i) c[i] = vkvref_bf16_to_f64(row[i]);
        uint16_t* out = index ? index + ru * index_stride : NULL;
        uint16_t dig[D_LAT];
        float e0, e1, e2, e3;
        project_and_bound(c, P, r, dig, &e0, &e3, &e1, &e2);
        if (out) {
            int off = 0;
            if (with_rope) {
                memcpy(out, row + D_LAT, D_ROPE * sizeof(uint16_t));
                off = D_ROPE;
            }
            memcpy(out + off, dig, (size_t)r * sizeof(uint16_t));
        }
        if (eta) {
            eta[ru] = e0;
            eps[ru] = e1;
            gam[ru] = e2;
        }
    }
    return 0;
}

/* Query side of the index score: the index-space query of each head,
 *   qt[b,h,:] = [ q_rope (mode has rope) ; RNE_bf16(P q_lat) (mode has digest) ]
 * and the head certificate scalars (a_h, n_h, e_h) used by the bound.
 * mode: 1 = rope only, 2 = digest only, 3 = rope + digest. */
int vkvref_query_prep(const uint16_t* q_lat, const uint16_t* q_rope, int64_t B, int64_t H,
                      const uint16_t* P, int r, int mode, uint16_t* qt, float* a, float* nq,
                      float* e) {
    int n = ((mode & 1) ? D_ROPE : 0) + ((mode & 2) ? r : 0);
    for (int64_t bh = 0; bh < B * H; ++bh) {
        double q[D_LAT];
        for (int i = 0; i < D_LAT; ++i) q[i] = vkvref_bf16_to_f64(q_lat[bh * D_LAT + i]);
        uint16_t dig[D_LAT];
        float s_resid, s_dn, s_derr, s_pn;
        project_and_bound(q, P, r, dig, &s_resid, &s_dn, &s_derr, &s_pn);
        uint16_t* o = qt + bh * n;
        int off = 0;
        if (mode & 1) {
            memcpy(o, q_rope + bh * D_ROPE, D_ROPE * sizeof(uint16_t));
            off = D_ROPE;
        }
        if (mode & 2) memcpy(o + off, dig, (size_t)r * sizeof(uint16_t));
        if (a) {
            a[bh] = s_resid;
            nq[bh] = s_dn;
            e[bh] = s_derr;
        }
    }
    return 0;
}

/* --------------------------------------------------------- index scores */

/* key_u = max_h sum_d qt[h,d] * x_u[d] for archived rows u in [0, A):
 * the trigger's exact-branch and sketch terms (the positive scale lambda is
 * dropped: it does not change the ranking).  fp64, d ascending, from +0.
 * Also returns, if dd_mismatch is non-null, the number of (u,h) whose plain
 * fp64 sum differs from a compensated (double-double) sum: zero means every
 * key is the exact real dot product. */
int vkvref_index_keys(const uint16_t* qt, int64_t H, int n, const uint16_t* x,
                      int64_t x_stride, int64_t A, double* key, int64_t* dd_mismatch,
                      int nthreads) {
    int64_t bad = 0;
    double* q = (double*)malloc(sizeof(double) * (size_t)(H * n));
    for (int64_t i = 0; i < H * n; ++i) q[i] = vkvref_bf16_to_f64(qt[i]);
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(static) reduction(+ : bad)
#endif
    for (int64_t u = 0; u < A; ++u) {
        double xv[D_ROW];
        for (int d = 0; d < n; ++d) xv[d] = vkvref_bf16_to_f64(x[u * x_stride + d]);
        double best = -INFINITY;
        for (int64_t h = 0; h < H; ++h) {
            const double* qh = q + h * n;
            double acc = 0.0;
            for (int d = 0; d < n; ++d) acc = fma(qh[d], xv[d], acc);
            if (dd_mismatch) {
                /* TwoSum of every partial sum (products are exact): when no
                 * step has a rounding error the fp64 sum is the exact sum */
                double hi = 0.0;
                int inexact = 0;
                for (int d = 0; d < n; ++d) {
                    double p = qh[d] * xv[d];
                    double s = hi + p;
                    double bp = s - hi;
                    double err = (hi - (s - bp)) + (p - bp);
                    hi = s;
                    if (err != 0.0) inexact = 1;
                }
                if (inexact || hi != acc) bad += 1;
            }
            if (acc > best) best = acc;
        }
        key[u] = best;
    }
    free(q);
    if (dd_mismatch) *dd_mismatch = bad;
    return 0;
}

/* ---------------------------------------------------------------- top-k */

typedef struct {
    double key;
    int32_t idx;
} kv_t;

static int cmp_desc(const void* pa, const void* pb) {
    const kv_t* a = (const kv_t*)pa;
    const kv_t* b = (const kv_t*)pb;
    if (a->key > b->key) return -1;
    if (a->key < b->key) return 1;
    return (a->idx < b->idx) ? -1 : (a->idx > b->idx);
}

static int cmp_int(const void* pa, const void* pb) {
    int32_t a = *(const int32_t*)pa, b = *(const int32_t*)pb;
    return (a > b) - (a < b);
}

/* S = the first k rows of [0, A) ordered by (key desc, index asc), written
 * ascending; theta = min key over S (-inf when k = 0). */
int vkvref_select(const double* key, int64_t A, int64_t k, int32_t* sel, double* theta) {
    if (k < 0 || k > A) return -1;
    kv_t* v = (kv_t*)malloc(sizeof(kv_t) * (size_t)(A > 0 ? A : 1));
    for (int64_t u = 0; u < A; ++u) {
        v[u].key = key[u];
        v[u].idx = (int32_t)u;
    }
    qsort(v, (size_t)A, sizeof(kv_t), cmp_desc);
    double th = -INFINITY;
    for (int64_t i = 0; i < k; ++i) {
        sel[i] = v[i].idx;
        th = v[i].key;
    }
    qsort(sel, (size_t)k, sizeof(int32_t), cmp_int);
    *theta = th;
    free(v);
    return 0;
}

/* ------------------------------------------------------- bound / admit */

/* UB_u = max_h fl64( s^_h(u) + B_h(u) ),
 * B_h(u) = a'_h*eta_u + n_h*eps_u + e_h*gamma_u  evaluated as
 *          fma(a'_h, eta_u, fma(n_h, eps_u, e_h*gamma_u))  in fp64,
 * with s^_h(u) the index score of head h (as in vkvref_index_keys) and
 * a'_h = ru_f32(cert_mult * a_h) (the product of two floats is exact in fp64).
 * cert_mult is z / sqrt(d_c - r) of Eq. (trigger): cert_mult = 1 is the sound
 * Cauchy-Schwarz bound, for which |s_h(u) - s^_h(u)| <= B_h(u) is Lemma (Index
 * certificate) plus the bf16 rounding of the stored sketch, so UB_u bounds
 * the exact full score; cert_mult < 1 is the calibrated trigger, which scales
 * only the sketch-residual term (the rounding terms stay rigorous). */
int vkvref_upper_bounds(const uint16_t* qt, int64_t H, int n, const float* a, const float* nq,
                        const float* e, const uint16_t* x, int64_t x_stride, const float* eta,
                        const float* eps, const float* gam, int64_t A, double cert_mult, double* ub,
                        int nthreads) {
    double* q = (double*)malloc(sizeof(double) * (size_t)(H * n));
    float* as = (float*)malloc(sizeof(float) * (size_t)(H > 0 ? H : 1));
    for (int64_t i = 0; i < H * n; ++i) q[i] = vkvref_bf16_to_f64(qt[i]);
    for (int64_t h = 0; h < H; ++h) as[h] = vkvref_ru_f32(cert_mult * (double)a[h]);
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(static)
#endif
    for (int64_t u = 0; u < A; ++u) {
        double xv[D_ROW];
        for (int d = 0; d < n; ++d) xv[d] = vkvref_bf16_to_f64(x[u * x_stride + d]);
        double best = -INFINITY;
        for (int64_t h = 0; h < H; ++h) {
            const double* qh = q + h * n;
            double acc = 0.0;
            for (int d = 0; d < n; ++d) acc = fma(qh[d], xv[d], acc);
            double bh = fma((double)as[h], (double)eta[u],
                            fma((double)nq[h], (double)eps[u], (double)e[h] * (double)gam[u]));
            double t = acc + bh;
            if (t > best) best = t;
        }
        ub[u] = best;
    }
    free(as);
    free(q);
    return 0;
}

/* Admitted set (two-tier mode): rows u in [0, A) not in S with UB_u > theta,
 * ascending.  Returns the number of admitted rows; writes at most cap. */
int64_t vkvref_admit(const double* ub, int64_t A, const int32_t* sel, int64_t k, double theta,
                     int32_t* adm, int64_t cap) {
    char* in = (char*)calloc((size_t)(A > 0 ? A : 1), 1);
    for (int64_t i = 0; i < k; ++i) in[sel[i]] = 1;
    int64_t cnt = 0;
    for (int64_t u = 0; u < A; ++u) {
        if (in[u]) continue;
        if (ub[u] > theta) {
            if (cnt < cap) adm[cnt] = (int32_t)u;
            ++cnt;
        }
    }
    free(in);
    return cnt;
}

/* ------------------------------------------------ calibrated trigger (z) */

/* The conformal quantile of Sec. 4.2 (the z paragraph) with the closed-form
 * chain of Sec. 5.2 (Recommended configuration), from the single recall
 * target tau = tau_num / tau_den (a rational, so that the integer quantities
 * below are exact):
 *   alpha    = (1 - tau) / 2                 the gate's false-close budget
 *   tau_s    = tau / (1 - alpha) = 2 tau_num / (tau_den + tau_num)
 *   min_hard = ceil(tau_s / (1 - tau_s)) = ceil(2 tau_num / (tau_den - tau_num))
 *   k        = ceil((n + 1) tau_s)           1-based rank in the sorted zq
 *   z        = zq_(k), clamped to [0, zmax]
 * With fewer than min_hard hard calibration queries (or k > n) the quantile
 * does not exist and z = zmax (reading: the conservative end of the clamp).
 * Returns 0 and writes z, min_hard and k (k = 0 when z is the clamp). */
int vkvref_conformal_z(const double* zq, int64_t n, int64_t tau_num, int64_t tau_den, double zmax, double* z,
                       int64_t* min_hard, int64_t* rank) {
    if (tau_num <= 0 || tau_den <= tau_num) return -1;
    const int64_t mh = (2 * tau_num + (tau_den - tau_num) - 1) / (tau_den - tau_num);
    const int64_t k = ((n + 1) * 2 * tau_num + (tau_den + tau_num) - 1) / (tau_den + tau_num);
    *min_hard = mh;
    if (n < mh || k > n || k < 1) {
        *z = zmax;
        *rank = 0;
        return 0;
    }
    double* v = (double*)malloc(sizeof(double) * (size_t)n);
    memcpy(v, zq, sizeof(double) * (size_t)n);
    /* insertion sort: n is a calibration window (tens to a few thousand) */
    for (int64_t i = 1; i < n; ++i) {
        double x = v[i];
        int64_t j = i - 1;
        while (j >= 0 && v[j] > x) {
            v[j + 1] = v[j];
            --j;
        }
        v[j + 1] = x;
    }
    double q = v[k - 1];
    free(v);
    if (q > zmax) q = zmax;
    if (!(q > 0.0)) q = 0.0;   /* reading: an inflation, never a deflation */
    *z = q;
    *rank = k;
    return 0;
}

/* Exact full score of one row for one head (Sec. 3, Eq. (setup), unscaled):
 * latent dims 0..511 then branch dims 0..63, fp64 sequential from +0. */
static double full_score(const uint16_t* ql, const uint16_t* qr, const uint16_t* row) {
    double acc = 0.0;
    for (int i = 0; i < D_LAT; ++i) acc = fma(vkvref_bf16_to_f64(ql[i]), vkvref_bf16_to_f64(row[i]), acc);
    for (int i = 0; i < D_ROPE; ++i) acc = fma(vkvref_bf16_to_f64(qr[i]), vkvref_bf16_to_f64(row[D_LAT + i]), acc);
    return acc;
}

/* Per head h: the maximum over the listed rows of the exact full score
 * s_h(u) and the row attaining it (ties: the lower row index).  With the
 * attended tier-1 rows this is the trigger threshold s*_h (the tier-1 max
 * logit of Sec. 4.2 and its figure); with every row of the context it gives
 * the causal argmax row of a calibration query.  N = 0: -inf and -1. */
int vkvref_row_max(const uint16_t* q_lat, const uint16_t* q_rope, int64_t H, const uint16_t* cache_seq,
                   int64_t row_stride, const int32_t* rows, int64_t N, double* smax, int32_t* argmax) {
    for (int64_t h = 0; h < H; ++h) {
        double best = -INFINITY;
        int32_t arg = -1;
        for (int64_t j = 0; j < N; ++j) {
            const int32_t u = rows[j];
            const double s = full_score(q_lat + h * D_LAT, q_rope + h * D_ROPE, cache_seq + (int64_t)u * row_stride);
            if (s > best || (s == best && u < arg)) {
                best = s;
                arg = u;
            }
        }
        smax[h] = best;
        argmax[h] = arg;
    }
    return 0;
}

/* Trigger margins of the archived rows (Eq. (trigger) against the tier-1
 * maximum, per head, fired if any head's bound exceeds its threshold):
 *   margin_u = max_h fl64( fl64(s^_h(u) + B_h(u)) - s*_h ),  B_h as in
 *   vkvref_upper_bounds with a'_h = ru_f32(cert_mult * a_h).
 * margin_u > 0 iff some head has UB_h(u) > s*_h (an fp64 difference of two
 * doubles is positive exactly when the first is larger). */
int vkvref_trigger_margins(const uint16_t* qt, int64_t H, int n, const float* a, const float* nq,
                           const float* e, const uint16_t* x, int64_t x_stride, const float* eta,
                           const float* eps, const float* gam, int64_t A, double cert_mult,
                           const double* smax, double* margin, int nthreads) {
    double* q = (double*)malloc(sizeof(double) * (size_t)(H * n));
    float* as = (float*)malloc(sizeof(float) * (size_t)(H > 0 ? H : 1));
    for (int64_t i = 0; i < H * n; ++i) q[i] = vkvref_bf16_to_f64(qt[i]);
    for (int64_t h = 0; h < H; ++h) as[h] = vkvref_ru_f32(cert_mult * (double)a[h]);
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(static)
#endif
    for (int64_t u = 0; u < A; ++u) {
        double xv[D_ROW];
        for (int d = 0; d < n; ++d) xv[d] = vkvref_bf16_to_f64(x[u * x_stride + d]);
        double best = -INFINITY;
        for (int64_t h = 0; h < H; ++h) {
            const double* qh = q + h * n;
            double acc = 0.0;
            for (int d = 0; d < n; ++d) acc = fma(qh[d], xv[d], acc);
            double bh = fma((double)as[h], (double)eta[u],
                            fma((double)nq[h], (double)eps[u], (double)e[h] * (double)gam[u]));
            double m = (acc + bh) - smax[h];
            if (m > best) best = m;
        }
        margin[u] = best;
    }
    free(as);
    free(q);
    return 0;
}

/* The fired set: rows of [0, A) outside S with margin > 0, ascending; with
 * topj > 0 only the topj of them with the largest margins (ties: the lower
 * row index) -- the optional budgeted cap of Sec. 4.3 / the appendix's
 * deployment specification.  Returns the number fired (after the cap);
 * writes at most cap rows. */
static int cmp_fire(const void* pa, const void* pb) {
    const kv_t* a = (const kv_t*)pa;
    const kv_t* b = (const kv_t*)pb;
    if (a->key > b->key) return -1;
    if (a->key < b->key) return 1;
    return (a->idx < b->idx) ? -1 : (a->idx > b->idx);
}

int64_t vkvref_fire(const double* margin, int64_t A, const int32_t* sel, int64_t k, int64_t topj, int32_t* fired,
                    int64_t cap) {
    char* in = (char*)calloc((size_t)(A > 0 ? A : 1), 1);
    for (int64_t i = 0; i < k; ++i) in[sel[i]] = 1;
    kv_t* v = (kv_t*)malloc(sizeof(kv_t) * (size_t)(A > 0 ? A : 1));
    int64_t nf = 0;
    for (int64_t u = 0; u < A; ++u)
        if (!in[u] && margin[u] > 0.0) {
            v[nf].key = margin[u];
            v[nf].idx = (int32_t)u;
            ++nf;
        }
    if (topj > 0 && nf > topj) {
        qsort(v, (size_t)nf, sizeof(kv_t), cmp_fire);
        nf = topj;
    }
    int32_t* out = (int32_t*)malloc(sizeof(int32_t) * (size_t)(nf > 0 ? nf : 1));
    for (int64_t i = 0; i < nf; ++i) out[i] = v[i].idx;
    qsort(out, (size_t)nf, sizeof(int32_t), cmp_int);
    for (int64_t i = 0; i < nf && i < cap; ++i) fired[i] = out[i];
    free(out);
    free(v);
    free(in);
    return nf;
}

/* Required inflation of one calibration query for head h (the z paragraph of
 * Sec. 4.2): with u* = the causal argmax row over the whole context,
 * the query is hard for h when u* is archived and outside the tier-1 set;
 * then z_q = (s*_h - idx_h(u*)) / cert_h(u*) with
 *   idx_h(u)  = fl64(s^_h(u) + fma(n_h, eps_u, e_h gam_u))   (the index score with its rounding slack)
 *   cert_h(u) = a_h eta_u / sqrt(d_c - r)                       (the per-dimension certificate scale)
 * so that the trigger score idx + z cert reaches s*_h exactly at z = z_q.
 * Writes hard[h] (0/1) and zq[h] (+inf when cert = 0 and s* > idx). */
int vkvref_required_inflation(const uint16_t* qt, int64_t H, int n, const float* a, const float* nq,
                              const float* e, const uint16_t* x, int64_t x_stride, const float* eta,
                              const float* eps, const float* gam, int64_t A, const int32_t* sel, int64_t k,
                              int r, const double* tier1_max, const int32_t* argmax, int32_t* hard, double* zq) {
    const double scale = sqrt((double)(D_LAT - r));
    for (int64_t h = 0; h < H; ++h) {
        const int32_t u = argmax[h];
        int in_s = 0;
        for (int64_t i = 0; i < k; ++i)
            if (sel[i] == u) in_s = 1;
        hard[h] = (u >= 0 && u < A && !in_s) ? 1 : 0;
        zq[h] = 0.0;
        if (!hard[h]) continue;
        double acc = 0.0;
        for (int d = 0; d < n; ++d)
            acc = fma(vkvref_bf16_to_f64(qt[h * n + d]), vkvref_bf16_to_f64(x[(int64_t)u * x_stride + d]), acc);
        const double idx = acc + fma((double)nq[h], (double)eps[u], (double)e[h] * (double)gam[u]);
        const double cert = (double)a[h] * (double)eta[u] / scale;
        const double gap = tier1_max[h] - idx;
        zq[h] = cert > 0.0 ? gap / cert : (gap > 0.0 ? INFINITY : -INFINITY);
    }
    return 0;
}

/* ---------------------------------------------------------------- attend */

/* Exact softmax attention of every head over the multiset of rows listed in
 * rows[0..N) of one sequence (Sec. 3, Eq. (setup); Lemma (Exchangeability)):
 *   s_h(u) = scale * ( q_lat[h].c_u + q_rope[h].r_u )      (576 dims, fp64)
 *   out[h] = sum_u exp(s_h(u) - m_h) c_u / sum_u exp(s_h(u) - m_h)
 *   lse[h] = m_h + log sum_u exp(s_h(u) - m_h)              (natural log)
 * The value is the 512-dim latent (the absorbed up-projection is applied
 * after attention, outside this path).  N = 0 gives out = 0, lse = -inf. */
int vkvref_attend(const uint16_t* q_lat, const uint16_t* q_rope, int64_t H,
                  const uint16_t* cache_seq, int64_t row_stride, const int32_t* rows, int64_t N,
                  double scale, double* out, double* lse, int nthreads) {
    double* s = (double*)malloc(sizeof(double) * (size_t)(N > 0 ? N : 1) * (size_t)H);
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(static)
#endif
    for (int64_t j = 0; j < N; ++j) {
        const uint16_t* row = cache_seq + (int64_t)rows[j] * row_stride;
        double c[D_ROW];
        for (int i = 0; i < D_ROW; ++i) c[i] = vkvref_bf16_to_f64(row[i]);
        for (int64_t h = 0; h < H; ++h) {
            double acc = 0.0;
            for (int i = 0; i < D_LAT; ++i)
                acc = fma(vkvref_bf16_to_f64(q_lat[h * D_LAT + i]), c[i], acc);
            for (int i = 0; i < D_ROPE; ++i)
                acc = fma(vkvref_bf16_to_f64(q_rope[h * D_ROPE + i]), c[D_LAT + i], acc);
            s[j * H + h] = scale * acc;
        }
    }
#ifdef _OPENMP
#pragma omp parallel for schedule(static)
#endif
    for (int64_t h = 0; h < H; ++h) {
        double* o = out + h * D_LAT;
        for (int i = 0; i < D_LAT; ++i) o[i] = 0.0;
        if (N == 0) {
            lse[h] = -INFINITY;
            continue;
        }
        double m = -INFINITY;
        for (int64_t j = 0; j < N; ++j)
            if (s[j * H + h] > m) m = s[j * H + h];
        double z = 0.0;
        for (int64_t j = 0; j < N; ++j) {
            double w = exp(s[j * H + h] - m);
            z += w;
            const uint16_t* row = cache_seq + (int64_t)rows[j] * row_stride;
            for (int i = 0; i < D_LAT; ++i) o[i] += w * vkvref_bf16_to_f64(row[i]);
        }
        for (int i = 0; i < D_LAT; ++i) o[i] /= z;
        lse[h] = m + log(z);
    }
    free(s);
    return 0;
}

/* Full archived-row scores s_h(u) (unscaled, 576 dims, fp64) for rows
 * [0, A): the quantity the certificate bounds.  Used by invariant tests. */
int vkvref_full_scores(const uint16_t* q_lat, const uint16_t* q_rope, int64_t H,
                       const uint16_t* cache_seq, int64_t row_stride, int64_t A, double* s,
                       int nthreads) {
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(static)
#endif
    for (int64_t u = 0; u < A; ++u) {
        const uint16_t* row = cache_seq + u * row_stride;
        for (int64_t h = 0; h < H; ++h) {
            double acc = 0.0;
            for (int i = 0; i < D_LAT; ++i)
                acc = fma(vkvref_bf16_to_f64(q_lat[h * D_LAT + i]), vkvref_bf16_to_f64(row[i]),
                          acc);
            for (int i = 0; i < D_ROPE; ++i)
                acc = fma(vkvref_bf16_to_f64(q_rope[h * D_ROPE + i]),
                          vkvref_bf16_to_f64(row[D_LAT + i]), acc);
            s[u * H + h] = acc;
        }
    }
    return 0;
}

/* ------------------------------------------------------ page-box bound */

/* Page-bound pruning (appendix "The dividend inside prior algorithms", the
 * page-bound paragraph and its equation): the archived rows [0, A) are cut
 * into pages of `page` consecutive rows (the last one ragged); the box of
 * page j is the per-column range of its index rows,
 *   lo_d = min_{u in page} x_u[d],   hi_d = max_{u in page} x_u[d],
 * written as bf16 bits (min and max of bf16 values are bf16 values; a zero
 * is written as +0).  Layout box[j][0][d] = lo, box[j][1][d] = hi. */
int vkvref_page_box(const uint16_t* x, int64_t x_stride, int n, int64_t A, int64_t page, uint16_t* box) {
    if (page < 1) return -1;
    const int64_t np = (A + page - 1) / page;
    for (int64_t j = 0; j < np; ++j) {
        const int64_t u0 = j * page, u1 = (u0 + page < A) ? u0 + page : A;
        for (int d = 0; d < n; ++d) {
            double lo = INFINITY, hi = -INFINITY;
            for (int64_t u = u0; u < u1; ++u) {
                const double v = vkvref_bf16_to_f64(x[u * x_stride + d]);
                if (v < lo) lo = v;
                if (v > hi) hi = v;
            }
            box[(j * 2 + 0) * n + d] = (lo == 0.0) ? 0 : vkvref_round_bf16(lo);
            box[(j * 2 + 1) * n + d] = (hi == 0.0) ? 0 : vkvref_round_bf16(hi);
        }
    }
    return 0;
}

/* The page's interval bound, maximised over heads:
 *   bound[j] = max_h sum_d max(qt[h,d] lo_d, qt[h,d] hi_d)
 * The larger of the two products is qt[h,d] hi_d when qt[h,d] >= 0 and
 * qt[h,d] lo_d otherwise, so each term is one product of bf16 values (exact
 * in fp64), summed d ascending from +0 with one rounding per term: the order
 * of the index key.  Every term is >= the key's term q_d x_u[d] for every row
 * u of the page and fp64 rounding is monotone, so bound[j] >= key_u for every
 * u in the page, bit for bit (the positive scale lambda is dropped as in the
 * keys). */
int vkvref_page_bound(const uint16_t* qt, int64_t H, int n, const uint16_t* box, int64_t npages, double* bound) {
    for (int64_t j = 0; j < npages; ++j) {
        const uint16_t* lo = box + (j * 2 + 0) * n;
        const uint16_t* hi = box + (j * 2 + 1) * n;
        double best = -INFINITY;
        for (int64_t h = 0; h < H; ++h) {
            double acc = 0.0;
            for (int d = 0; d < n; ++d) {
                const double q = vkvref_bf16_to_f64(qt[h * n + d]);
                const double e = (q >= 0.0) ? vkvref_bf16_to_f64(hi[d]) : vkvref_bf16_to_f64(lo[d]);
                acc = fma(q, e, acc);
            }
            if (acc > best) best = acc;
        }
        bound[j] = best;
    }
    return 0;
}

int vkvref_max_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
