/*
 * kan_oracle.c -- plain, slow, float64 reference for the InKAN KAN-layer
 * forward (B-spline KAN layer with the basis in clamped truncated-power form).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file: only the tests, the smoke check and the CPU-baseline leg of
 * the benchmark use it.  It shares no code, header, table or constant with the
 * HIP library; the two meet only through seeded inputs.
 *
 * Every routine below is a direct transcription of a definition in the paper,
 * evaluated in IEEE double with plain loops, no blocking and no reordering
 * beyond what the definition states:
 *
 *   knots            -- uniform simple knot vector (Sec. 2, Step 3), extended
 *                       by k spans on each side of [lo, hi] (reading of the
 *                       grid convention: t_j = lo + (j - k) h, j = 0..G+2k).
 *   basis_tp         -- truncated-power form (Sec. 2 Step 4, eq. general_truncated
 *                       and, for k = 3, eq. truncated) with the bounded
 *                       coordinate of Sec. 2 "Bounded-coordinate stabilization"
 *                       (eq. bounded), or without it (clamp = 0).
 *   basis_cdb        -- Cox-de Boor recursion (eq. cdb0, eq. cdbk).
 *   basis_seg        -- uniform cubic segment form T(tau) * M_B-spline
 *                       (eq. bspline_matrix), k = 3 only.
 *   layer            -- KAN layer forward (eq. kan_forward) with SiLU base
 *                       branch sigma(x) = x / (1 + exp(-x)).
 *   round_bf16       -- round-to-nearest-even to bfloat16 (8 significant
 *                       bits), used to mirror bf16 storage between layers.
 *   basis_tp_deriv   -- d N_{j,k} / dx of the clamped truncated-power form:
 *                       eq. general_truncated differentiated term by term
 *                       (power k - 1, factor k), times the derivative of the
 *                       clamp of eq. bounded (1 inside (0, k+1), else 0).
 *   layer_backward   -- gradients of eq. kan_forward for an upstream gradient
 *                       dy: dC = dy^T Phi(x), dWb = dy^T sigma(x), and
 *                       dx = sum_o dy (sum_j C N_j'(x) + Wb sigma'(x)).  The
 *                       paper times the forward only (Sec. 5 lists backward
 *                       timing as future work); these are the chain rule
 *                       applied to its forward.
 *
 * Build: gcc -O2 -fopenmp -fPIC -shared (no -ffast-math; the rounding of every
 * double operation must be IEEE).
 */
#include <math.h>
#include <stdint.h>
#include <stddef.h>
#include <omp.h>
#include <stdlib.h>

/* ---------------------------------------------------------------- helpers */

static double binom(int n, int r) {
    double c = 1.0;
    for (int i = 1; i <= r; ++i) c = c * (double)(n - r + i) / (double)i;
    return c;
}

static double factorial(int n) {
    double f = 1.0;
    for (int i = 2; i <= n; ++i) f *= (double)i;
    return f;
}

static double ipow(double v, int k) {
    double p = 1.0;
    for (int i = 0; i < k; ++i) p *= v;
    return p;
}

int kan_oracle_num_threads(void) { return omp_get_max_threads(); }
void kan_oracle_set_threads(int n) { if (n > 0) omp_set_num_threads(n); }

/* ------------------------------------------------------------------ knots */

/* Knot vector of a uniform grid of G intervals on [lo, hi] for degree k:
 * t_j = lo + (j - k) h, h = (hi - lo) / G, j = 0 .. G + 2k.  This gives
 * G + k basis functions N_0 .. N_{G+k-1}; basis j is supported on
 * [t_j, t_{j+k+1}], and [lo, hi] = [t_k, t_{G+k}].  t must hold G + 2k + 1. */
void kan_oracle_knots(int G, int k, double lo, double hi, double* t) {
    double h = (hi - lo) / (double)G;
    for (int j = 0; j <= G + 2 * k; ++j) t[j] = lo + (double)(j - k) * h;
}

/* ---------------------------------------------- truncated-power (O1) form */

/* N_{j,k}(x) = 1/(k! h^k) sum_{m=0}^{k+1} (-1)^m C(k+1, m) (x - t_{j+m})_+^k
 * (eq. general_truncated).  In the normalised coordinate u = (x - t_j)/h this
 * is (1/k!) sum_m (-1)^m C(k+1, m) (u - m)_+^k, which for k = 3 is eq. truncated
 * with the stencil {1, -4, 6, -4, 1} / 6.  With clamp != 0 the coordinate is
 * first bounded to [0, k+1] (eq. bounded).  A NaN input gives NaN (the clamp
 * must not swallow it). */
static void tp_row(double xv, int G, int k, double lo, double hi, int clamp,
                   double* row) {
    const int nb = G + k;
    const double h = (hi - lo) / (double)G;
    const double inv_kfact = 1.0 / factorial(k);
    for (int j = 0; j < nb; ++j) {
        if (isnan(xv)) { row[j] = xv; continue; }
        const double tj = lo + (double)(j - k) * h;
        double u = (xv - tj) / h;
        if (clamp) {
            if (u < 0.0) u = 0.0;
            if (u > (double)(k + 1)) u = (double)(k + 1);
        }
        double s = 0.0;
        for (int m = 0; m <= k + 1; ++m) {
            const double z = u - (double)m;
            const double zp = z > 0.0 ? z : 0.0;
            const double term = binom(k + 1, m) * ipow(zp, k);
            s += (m & 1) ? -term : term;
        }
        row[j] = s * inv_kfact;
    }
}

/* phi is [n, G + k], basis index fastest. */
void kan_oracle_basis_tp(const double* x, int64_t n, int G, int k, double lo,
                         double hi, int clamp, double* phi) {
    const int nb = G + k;
    #pragma omp parallel for schedule(static)
    for (int64_t e = 0; e < n; ++e)
        tp_row(x[e], G, k, lo, hi, clamp, &phi[e * nb]);
}

/* ------------------------------------------------- Cox-de Boor (O2) form */

/* N_{j,0}(x) = [t_j <= x < t_{j+1}] (eq. cdb0); for p = 1..k
 * N_{j,p} = (x - t_j)/(t_{j+p} - t_j) N_{j,p-1}
 *         + (t_{j+p+1} - x)/(t_{j+p+1} - t_{j+1}) N_{j+1,p-1}   (eq. cdbk).
 * With simple uniform knots every denominator is p*h > 0.  t holds the
 * G + 2k + 1 knots; work holds at least G + 2k doubles. */
static void cdb_row(double xv, int G, int k, const double* t, double* work,
                    double* row) {
    const int nb = G + k;
    const int nk = G + 2 * k + 1;
    if (isnan(xv)) {
        for (int j = 0; j < nb; ++j) row[j] = xv;
        return;
    }
    /* degree 0: one indicator per knot interval, nk - 1 of them */
    for (int j = 0; j < nk - 1; ++j)
        work[j] = (t[j] <= xv && xv < t[j + 1]) ? 1.0 : 0.0;
    for (int p = 1; p <= k; ++p) {
        /* ascending j reads work[j] and work[j + 1] before work[j] is replaced */
        for (int j = 0; j < nk - 1 - p; ++j) {
            const double a = (xv - t[j]) / (t[j + p] - t[j]);
            const double b = (t[j + p + 1] - xv) / (t[j + p + 1] - t[j + 1]);
            work[j] = a * work[j] + b * work[j + 1];
        }
    }
    for (int j = 0; j < nb; ++j) row[j] = work[j];
}

void kan_oracle_basis_cdb(const double* x, int64_t n, int G, int k, double lo,
                          double hi, double* phi) {
    const int nb = G + k;
    #pragma omp parallel
    {
        double* t = (double*)malloc(sizeof(double) * (size_t)(G + 2 * k + 1));
        double* work = (double*)malloc(sizeof(double) * (size_t)(G + 2 * k + 1));
        kan_oracle_knots(G, k, lo, hi, t);
        #pragma omp for schedule(static)
        for (int64_t e = 0; e < n; ++e) cdb_row(x[e], G, k, t, work, &phi[e * nb]);
        free(work);
        free(t);
    }
}

/* ------------------------------------------ cubic segment (O3) form, k=3 */

/* On the knot span [t_m, t_{m+1}) with local parameter tau in [0, 1), the four
 * nonzero cubic bases are [N_{m-3}, N_{m-2}, N_{m-1}, N_m] = [1 tau tau^2 tau^3]
 * * M_B-spline (eq. bspline_matrix); every other basis is 0.  Spans are
 * half-open, as in eq. cdb0, so x = t_{G+6} lies outside every support. */
void kan_oracle_basis_seg(const double* x, int64_t n, int G, double lo,
                          double hi, double* phi) {
    static const double M[4][4] = {
        { 1.0 / 6.0,  4.0 / 6.0,  1.0 / 6.0, 0.0 },
        {-3.0 / 6.0,  0.0,        3.0 / 6.0, 0.0 },
        { 3.0 / 6.0, -6.0 / 6.0,  3.0 / 6.0, 0.0 },
        {-1.0 / 6.0,  3.0 / 6.0, -3.0 / 6.0, 1.0 / 6.0 },
    };
    const int k = 3;
    const int nb = G + k;
    const double h = (hi - lo) / (double)G;
    const double t0 = lo - 3.0 * h;
    #pragma omp parallel for schedule(static)
    for (int64_t e = 0; e < n; ++e) {
        const double xv = x[e];
        for (int j = 0; j < nb; ++j) phi[e * nb + j] = 0.0;
        if (isnan(xv)) {
            for (int j = 0; j < nb; ++j) phi[e * nb + j] = xv;
            continue;
        }
        const double s = (xv - t0) / h;
        if (!(s >= 0.0) || s >= (double)(G + 2 * k)) continue; /* off all spans */
        const int m = (int)floor(s);
        const double tau = s - (double)m;
        const double T[4] = { 1.0, tau, tau * tau, tau * tau * tau };
        for (int c = 0; c < 4; ++c) {
            const int j = m - 3 + c;
            if (j < 0 || j >= nb) continue;
            double v = 0.0;
            for (int r = 0; r < 4; ++r) v += T[r] * M[r][c];
            phi[e * nb + j] = v;
        }
    }
}

/* ----------------------------------------------------------------- SiLU */

/* sigma(x) = x * sigmoid(x) = x / (1 + exp(-x)), the base function of the
 * residual branch in eq. kan_forward. */
static double silu_one(double v) { return v / (1.0 + exp(-v)); }

void kan_oracle_silu(const double* x, int64_t n, double* out) {
    #pragma omp parallel for schedule(static)
    for (int64_t e = 0; e < n; ++e) out[e] = silu_one(x[e]);
}

void kan_oracle_round_bf16(const double* v, int64_t n, double* out);

/* ------------------------------------------------------------ KAN layer */

/* y[b, o] = sum_i ( sum_j C[o, i, j] N_j(x[b, i]) + Wb[o, i] sigma(x[b, i]) )
 * (eq. kan_forward), with N from the truncated-power form (basis_kind 0,
 * clamped) or the Cox-de Boor recursion (basis_kind 1).  x is [B, in],
 * C is [out, in, G + k], Wb is [out, in], y is [B, out]; all row-major.
 * For each output the sum runs over i, and within i over j then the SiLU
 * term, in index order, accumulated in double.  With bf16_operands != 0 every
 * basis value and every SiLU value is rounded to bfloat16 before it enters the
 * contraction (the operands a bf16 matrix unit consumes); the products and
 * sums stay in double. */
void kan_oracle_layer(const double* x, int64_t B, int in, int out,
                      const double* C, const double* Wb, int G, int k,
                      double lo, double hi, int basis_kind, int bf16_operands,
                      double* y) {
    const int nb = G + k;
    #pragma omp parallel
    {
        double* t = (double*)malloc(sizeof(double) * (size_t)(G + 2 * k + 1));
        double* work = (double*)malloc(sizeof(double) * (size_t)(G + 2 * k + 1));
        double* nrow = (double*)malloc(sizeof(double) * (size_t)in * (size_t)nb);
        double* sg = (double*)malloc(sizeof(double) * (size_t)in);
        kan_oracle_knots(G, k, lo, hi, t);
        #pragma omp for schedule(dynamic, 1)
        for (int64_t b = 0; b < B; ++b) {
            const double* xb = &x[b * (int64_t)in];
            for (int i = 0; i < in; ++i) {
                if (basis_kind == 1)
                    cdb_row(xb[i], G, k, t, work, &nrow[(int64_t)i * nb]);
                else
                    tp_row(xb[i], G, k, lo, hi, 1, &nrow[(int64_t)i * nb]);
                sg[i] = silu_one(xb[i]);
                if (bf16_operands) {
                    kan_oracle_round_bf16(&nrow[(int64_t)i * nb], nb, &nrow[(int64_t)i * nb]);
                    kan_oracle_round_bf16(&sg[i], 1, &sg[i]);
                }
            }
            for (int o = 0; o < out; ++o) {
                double s = 0.0;
                for (int i = 0; i < in; ++i) {
                    const double* c = &C[((int64_t)o * in + i) * nb];
                    const double* nr = &nrow[(int64_t)i * nb];
                    for (int j = 0; j < nb; ++j) s += c[j] * nr[j];
                    s += Wb[(int64_t)o * in + i] * sg[i];
                }
                y[b * (int64_t)out + o] = s;
            }
        }
        free(sg);
        free(nrow);
        free(work);
        free(t);
    }
}

/* ------------------------------------------------------- bf16 rounding */

/* Round each double to the nearest bfloat16 value (8 significant bits, 8-bit
 * exponent), ties to even, and return it as a double.  Values beyond the
 * largest finite bf16 after rounding become +-inf; NaN stays NaN; results below
 * the normal range are rounded on the subnormal grid 2^-133. */
void kan_oracle_round_bf16(const double* v, int64_t n, double* out) {
    for (int64_t e = 0; e < n; ++e) {
        const double a = v[e];
        if (isnan(a) || isinf(a) || a == 0.0) { out[e] = a; continue; }
        int ex;
        frexp(a, &ex);                 /* |a| in [2^(ex-1), 2^ex) */
        int q = ex - 8;                /* quantum exponent for 8 significant bits */
        if (q < -133) q = -133;        /* bf16 subnormal spacing */
        const double scaled = ldexp(a, -q);
        const double r = nearbyint(scaled); /* default mode: ties to even */
        double res = ldexp(r, q);
        if (fabs(res) > 3.3895313892515355e38) res = a > 0 ? INFINITY : -INFINITY;
        out[e] = res;
    }
}

/* ------------------------------------------------------------ backward */

/* d/dx of the clamped basis N_j at x.  Differentiating eq. general_truncated
 * in x gives (1 / ((k-1)! h^k)) sum_m (-1)^m C(k+1, m) (x - t_{j+m})_+^{k-1},
 * i.e. (1/h) (1/(k-1)!) sum_m (-1)^m C(k+1, m) (u - m)_+^{k-1} in u; with
 * the clamp of eq. bounded the form is N(ubar(u)), whose derivative is that
 * sum at ubar times dubar/du = [0 < u < k+1].  (z)_+^0 is read as [z > 0].
 * A NaN input gives NaN. */
static void tp_deriv_row(double xv, int G, int k, double lo, double hi, double* row) {
    const int nb = G + k;
    const double h = (hi - lo) / (double)G;
    const double inv_fact = 1.0 / factorial(k - 1);
    for (int j = 0; j < nb; ++j) {
        if (isnan(xv)) { row[j] = xv; continue; }
        const double tj = lo + (double)(j - k) * h;
        const double u = (xv - tj) / h;
        if (!(u > 0.0 && u < (double)(k + 1))) { row[j] = 0.0; continue; }
        double s = 0.0;
        for (int m = 0; m <= k + 1; ++m) {
            const double z = u - (double)m;
            const double zp = (k - 1 == 0) ? (z > 0.0 ? 1.0 : 0.0) : ipow(z > 0.0 ? z : 0.0, k - 1);
            const double term = binom(k + 1, m) * zp;
            s += (m & 1) ? -term : term;
        }
        row[j] = s * inv_fact / h;
    }
}

void kan_oracle_basis_tp_deriv(const double* x, int64_t n, int G, int k, double lo,
                               double hi, double* dphi) {
    const int nb = G + k;
    #pragma omp parallel for schedule(static)
    for (int64_t e = 0; e < n; ++e)
        tp_deriv_row(x[e], G, k, lo, hi, &dphi[e * nb]);
}

/* sigma'(x) for sigma(x) = x / (1 + exp(-x)): with s = 1 / (1 + exp(-x)),
 * d(x s)/dx = s + x s (1 - s). */
static double silu_deriv_one(double v) {
    const double s = 1.0 / (1.0 + exp(-v));
    return s + v * s * (1.0 - s);
}

void kan_oracle_silu_deriv(const double* x, int64_t n, double* out) {
    #pragma omp parallel for schedule(static)
    for (int64_t e = 0; e < n; ++e) out[e] = silu_deriv_one(x[e]);
}

/* Gradients of L = sum_{b,o} dy[b, o] y[b, o] with y from eq. kan_forward:
 *   dx[b, i]  = sum_o dy[b, o] ( sum_j C[o, i, j] N_j'(x[b, i]) + Wb[o, i] sigma'(x[b, i]) )
 *   dC[o,i,j] = sum_b dy[b, o] N_j(x[b, i])
 *   dWb[o, i] = sum_b dy[b, o] sigma(x[b, i])
 * x [B, in], C [out, in, G + k], Wb [out, in], dy [B, out]; outputs dx
 * [B, in], dC [out, in, G + k], dWb [out, in].  Plain loops in double, each
 * sum in index order (o, then j; b ascending). */
void kan_oracle_layer_backward(const double* x, int64_t B, int in, int out,
                               const double* C, const double* Wb, const double* dy,
                               int G, int k, double lo, double hi,
                               double* dx, double* dC, double* dWb) {
    const int nb = G + k;
    /* dx: rows are independent */
    #pragma omp parallel
    {
        double* dn = (double*)malloc(sizeof(double) * (size_t)nb);
        #pragma omp for schedule(dynamic, 4)
        for (int64_t b = 0; b < B; ++b) {
            for (int i = 0; i < in; ++i) {
                const double xv = x[b * (int64_t)in + i];
                tp_deriv_row(xv, G, k, lo, hi, dn);
                const double sd = silu_deriv_one(xv);
                double s = 0.0;
                for (int o = 0; o < out; ++o) {
                    const double g = dy[b * (int64_t)out + o];
                    const double* c = &C[((int64_t)o * in + i) * nb];
                    double t = 0.0;
                    for (int j = 0; j < nb; ++j) t += c[j] * dn[j];
                    t += Wb[(int64_t)o * in + i] * sd;
                    s += g * t;
                }
                dx[b * (int64_t)in + i] = s;
            }
        }
        free(dn);
    }
    /* dC, dWb: one (o, i) pair per iteration, the sum over b in order */
    #pragma omp parallel
    {
        double* nrow = (double*)malloc(sizeof(double) * (size_t)nb);
        double* acc = (double*)malloc(sizeof(double) * (size_t)nb);
        #pragma omp for schedule(dynamic, 1) collapse(2)
        for (int o = 0; o < out; ++o) {
            for (int i = 0; i < in; ++i) {
                double accw = 0.0;
                for (int j = 0; j < nb; ++j) acc[j] = 0.0;
                for (int64_t b = 0; b < B; ++b) {
                    const double g = dy[b * (int64_t)out + o];
                    const double xv = x[b * (int64_t)in + i];
                    tp_row(xv, G, k, lo, hi, 1, nrow);
                    for (int j = 0; j < nb; ++j) acc[j] += g * nrow[j];
                    accw += g * silu_one(xv);
                }
                for (int j = 0; j < nb; ++j) dC[((int64_t)o * in + i) * nb + j] = acc[j];
                dWb[(int64_t)o * in + i] = accw;
            }
        }
        free(acc);
        free(nrow);
    }
}
