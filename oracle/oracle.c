/*
 * oracle.c -- fp64 CPU oracle for the gated N-D FFT long convolution.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file; only the tests, the smoke check and the benchmark's CPU
 * baseline do.  It shares no code, header, table or helper with the HIP
 * library.
 *
 * What it computes (paper: Def. A.2 "Hyena mixer" with its shortcut vector,
 * Def. A.3 "Gated Hyena mixer", and the HyenaND operator, Eq. (HyenaND) of
 * section 3.2, restricted to the long convolution and its two gates):
 *
 *   u = x1 * v                                   (inner gate, elementwise)
 *   linear:   conv[n] = sum_{m : 0 <= m_d <= n_d}  k[m] u[n - m]
 *   circular: conv[n] = sum_{m in box}            k[m] u[(n - m) mod L]
 *   centered: conv[n] = sum_{m in box}            kc[n - m + (L - 1)] u[m]
 *   y[n]     = x2[n] * (conv[n] + D[c] u[n])     (shortcut, then outer gate)
 *
 * for every sample b, channel c and output index n of the L1 x ... x LN grid,
 * with k[b, c] the sample's own kernel (section 3.2.2, "FFT path
 * preservation": one kernel per input).  "linear" is the non-circular
 * convolution of section 3.2.1 ("Support for circular and non-circular
 * convolutions"): zero-pad and crop, with index 0 of k the zero displacement;
 * "circular" treats the grid as a torus.  "centered" is the same section's
 * kernel on the double grid: kc has 2 L_d - 1 points per axis, index L_d - 1
 * is the zero displacement, so every displacement -(L_d - 1) .. L_d - 1
 * between two points of the input grid has its own weight; the input is
 * zero-padded to 2 L_d and the output cropped to the first L_d.  kc is
 * [B, C, 2 L1 - 1, ..., 2 LN - 1].
 *
 * Two independent evaluations are provided:
 *   oracle_direct / oracle_direct_points : the sum above written out.
 *   oracle_fft                          : the convolution theorem with this
 *       file's own iterative radix-2 FFT, transform size 2 L_d per axis in
 *       linear mode (the appendix "Hardware Context and IO Profile" requires a
 *       transform length of at least 2L-1 and uses about 2L) and L_d in
 *       circular mode, forward unnormalised, inverse scaled by 1/prod(P).
 *
 * All arithmetic is IEEE double.  Inputs arrive already upcast to double.
 * Layout: every tensor is contiguous row-major [B, C, L1, ..., LN]; D is [C].
 * dims = {B, C, L1, ..., LN}, ndim = N in {1, 2, 3}.
 *
 * Backward (gradients of a scalar loss through y; the derivatives of the
 * definition above, written out -- the paper trains HyenaND end to end through
 * this operator but prints no backward formulas): with gy = dLoss/dy,
 *
 *   z   = conv + D[c] u                 (pre-gate output)
 *   gx2 = gy * z
 *   h   = gy * x2                       (dLoss/dz)
 *   gu[j] = sum_n k[n - j] h[n] + D[c] h[j]      (adjoint of u -> k * u;
 *           linear: n_d >= j_d, n_d < L_d; circular: (n - j) mod L)
 *   gk[m] = sum_n h[n] u[n - m]                  (linear: n_d >= m_d;
 *           circular: u[(n - m) mod L])
 *   gx1 = gu * v,  gv = gu * x1,  gD[c] = sum_{b, n} h[b,c,n] u[b,c,n]
 *
 *   oracle_backward_direct : these sums written out (any extents).
 *   oracle_backward_fft    : the same through this file's FFT: on the
 *       transform grid the adjoint of a convolution with k is the product
 *       with conj(K) (k real), so gu = crop(IFFT(conj(K) H)) + D h and
 *       gk = crop(IFFT(conj(U) H)); zero padding to 2 L_d makes the cyclic
 *       sums equal the linear ones on the cropped range.
 *
 * The mode argument: 0 linear, 1 circular, 2 centered (the FFT backward
 * takes 0 and 1; the direct backward all three, centred as
 *   gu[j] = sum_n kc[n - j + (L - 1)] h[n] + D[c] h[j],
 *   gk[i] = sum_n h[n] u[n - i + (L - 1)]  over n with that index on the grid,
 * kc and gk on the 2 L_d - 1 point grid).
 *
 * The HyenaND operator, Eq. (HyenaND) of section 3.2 (oracle_operator):
 * with q, kin, vin the three projections [B, C, L...], per sample b and grid
 * point p, the channel vectors are normalised across the C channels:
 *
 *   a[c]  = q[c] / max(||q[:]||_2, eps_l2) * SiLU(kin[c])   (l2 norm of q)
 *   u[c]  = a[c] / sqrt(mean_c a^2 + eps_rms) * w_in[c]      (RMSNorm)
 *   z     = Sigmoid(vin) * (conv(k, u) + D[c] u)             (long conv,
 *           shortcut and outer gate; conv in the given mode)
 *   y[c]  = z[c] / sqrt(mean_c z^2 + eps_rms) * w_out[c]     (RMSNorm)
 *
 * with SiLU(x) = x / (1 + exp(-x)), Sigmoid(x) = 1 / (1 + exp(-x)).  The
 * paper writes the operator without the shortcut; D = 0 gives it exactly.
 *
 * Return codes: 0 ok, 1 bad argument, 2 out of memory, 3 the inverse
 * transform left an imaginary residue above 1e-9 of the real part (a broken
 * FFT), 4 a thread could not be started.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifndef M_PI
#define M_PI 3.14159265358979323846
#endif

typedef struct {
    double re, im;
} cplx;

typedef struct {
    int64_t B, C;
    int64_t L[3]; /* grid extents, padded to 3 axes with leading 1s */
    int64_t box;  /* prod L */
    int ndim;     /* number of real axes: the last ndim of L[] */
} geom;

static int make_geom(int ndim, const int64_t *dims, geom *g) {
    if (ndim < 1 || ndim > 3 || !dims) return 1;
    g->B = dims[0];
    g->C = dims[1];
    if (g->B < 1 || g->C < 1) return 1;
    for (int d = 0; d < 3; ++d) g->L[d] = 1;
    for (int d = 0; d < ndim; ++d) {
        if (dims[2 + d] < 1) return 1;
        g->L[3 - ndim + d] = dims[2 + d];
    }
    g->box = g->L[0] * g->L[1] * g->L[2];
    g->ndim = ndim;
    return 0;
}

enum { MODE_LINEAR = 0, MODE_CIRCULAR = 1, MODE_CENTERED = 2 };

/* Transform extents: in linear and centered mode the smallest power of two
 * >= 2 L_d - 1 on the real axes (2 L_d when L_d is a power of two; any length
 * >= 2 L_d - 1 holds every displacement between two grid points without
 * wrap-around), L_d in circular mode; the virtual leading axes of a 1D/2D
 * problem stay at extent 1. */
static int64_t pow2_at_least(int64_t n) {
    int64_t p = 1;
    while (p < n) p *= 2;
    return p;
}

static void transform_extents(const geom *g, int mode, int64_t P[3]) {
    for (int d = 0; d < 3; ++d) {
        int real_axis = d >= 3 - g->ndim;
        if (real_axis && mode != MODE_CIRCULAR)
            P[d] = g->L[d] > 1 ? pow2_at_least(2 * g->L[d] - 1) : 2;
        else
            P[d] = g->L[d];
    }
}

/* Points of the centered kernel per line: prod (2 L_d - 1) (1 on the virtual
 * axes). */
static int64_t centered_box(const geom *g) {
    return (2 * g->L[0] - 1) * (2 * g->L[1] - 1) * (2 * g->L[2] - 1);
}

/* ------------------------------------------------------------------------- */
/* Direct evaluation of the definition                                        */
/* ------------------------------------------------------------------------- */

/* One output element of line `line` (= b*C + c) at grid index (n0,n1,n2). */
static double direct_one(const double *x1, const double *x2, const double *v,
                         const double *k, const double *D, const geom *g,
                         int mode, int64_t line, int64_t n0, int64_t n1,
                         int64_t n2) {
    const int64_t L0 = g->L[0], L1 = g->L[1], L2 = g->L[2];
    const int64_t base = line * g->box;
    const double *X1 = x1 + base, *V = v + base, *K = k + base;
    double conv = 0.0;
    if (mode == MODE_CENTERED) {
        const int64_t K1 = 2 * L1 - 1, K2 = 2 * L2 - 1;
        const double *KC = k + line * centered_box(g);
        for (int64_t m0 = 0; m0 < L0; ++m0)
            for (int64_t m1 = 0; m1 < L1; ++m1)
                for (int64_t m2 = 0; m2 < L2; ++m2) {
                    int64_t j0 = n0 - m0 + L0 - 1, j1 = n1 - m1 + L1 - 1, j2 = n2 - m2 + L2 - 1;
                    int64_t un = (m0 * L1 + m1) * L2 + m2;
                    conv += KC[(j0 * K1 + j1) * K2 + j2] * (X1[un] * V[un]);
                }
    } else if (mode == MODE_LINEAR) {
        for (int64_t m0 = 0; m0 <= n0; ++m0)
            for (int64_t m1 = 0; m1 <= n1; ++m1)
                for (int64_t m2 = 0; m2 <= n2; ++m2) {
                    int64_t km = (m0 * L1 + m1) * L2 + m2;
                    int64_t un = ((n0 - m0) * L1 + (n1 - m1)) * L2 + (n2 - m2);
                    conv += K[km] * (X1[un] * V[un]);
                }
    } else {
        for (int64_t m0 = 0; m0 < L0; ++m0)
            for (int64_t m1 = 0; m1 < L1; ++m1)
                for (int64_t m2 = 0; m2 < L2; ++m2) {
                    int64_t km = (m0 * L1 + m1) * L2 + m2;
                    int64_t i0 = (n0 - m0 + L0) % L0;
                    int64_t i1 = (n1 - m1 + L1) % L1;
                    int64_t i2 = (n2 - m2 + L2) % L2;
                    int64_t un = (i0 * L1 + i1) * L2 + i2;
                    conv += K[km] * (X1[un] * V[un]);
                }
    }
    const int64_t c = line % g->C;
    const int64_t nn = (n0 * L1 + n1) * L2 + n2;
    const double u = X1[nn] * V[nn];
    return x2[base + nn] * (conv + D[c] * u);
}

typedef struct {
    const double *x1, *x2, *v, *k, *D;
    double *y;
    const geom *g;
    int circular; /* the mode: MODE_LINEAR, MODE_CIRCULAR or MODE_CENTERED */
    /* work split */
    const int64_t *items; /* line ids (direct/fft) or flat output indices (points) */
    int64_t nitems;
    int tid, nthreads;
    int status;
    /* fft-only shared tables */
    const cplx *const *tw_fwd; /* per axis: P_d/2 twiddles exp(-2 pi i j / P_d) */
    const cplx *const *tw_inv; /* per axis: P_d/2 twiddles exp(+2 pi i j / P_d) */
} job;

static int64_t item_at(const job *J, int64_t i) { return J->items ? J->items[i] : i; }

static void *direct_lines_worker(void *arg) {
    job *J = (job *)arg;
    const geom *g = J->g;
    for (int64_t i = J->tid; i < J->nitems; i += J->nthreads) {
        int64_t line = item_at(J, i);
        double *Y = J->y + line * g->box;
        for (int64_t n0 = 0; n0 < g->L[0]; ++n0)
            for (int64_t n1 = 0; n1 < g->L[1]; ++n1)
                for (int64_t n2 = 0; n2 < g->L[2]; ++n2)
                    Y[(n0 * g->L[1] + n1) * g->L[2] + n2] =
                        direct_one(J->x1, J->x2, J->v, J->k, J->D, g, J->circular, line, n0, n1, n2);
    }
    return NULL;
}

static void *direct_points_worker(void *arg) {
    job *J = (job *)arg;
    const geom *g = J->g;
    for (int64_t i = J->tid; i < J->nitems; i += J->nthreads) {
        int64_t flat = J->items[i];
        int64_t line = flat / g->box;
        int64_t r = flat % g->box;
        int64_t n2 = r % g->L[2];
        int64_t n1 = (r / g->L[2]) % g->L[1];
        int64_t n0 = r / (g->L[2] * g->L[1]);
        J->y[i] = direct_one(J->x1, J->x2, J->v, J->k, J->D, g, J->circular, line, n0, n1, n2);
    }
    return NULL;
}

static int run_jobs(job *proto, int nthreads, void *(*fn)(void *)) {
    if (nthreads < 1) nthreads = 1;
    if (nthreads > 256) nthreads = 256;
    job jobs[256];
    pthread_t th[256];
    int started[256];
    int rc = 0;
    for (int t = 0; t < nthreads; ++t) {
        jobs[t] = *proto;
        jobs[t].tid = t;
        jobs[t].nthreads = nthreads;
        jobs[t].status = 0;
        started[t] = 0;
    }
    for (int t = 1; t < nthreads; ++t) {
        if (pthread_create(&th[t], NULL, fn, &jobs[t]) == 0)
            started[t] = 1;
        else
            rc = 4;
    }
    fn(&jobs[0]);
    for (int t = 1; t < nthreads; ++t)
        if (started[t]) pthread_join(th[t], NULL);
    if (rc) return rc;
    for (int t = 0; t < nthreads; ++t)
        if (jobs[t].status) return jobs[t].status;
    return 0;
}

int oracle_direct(const double *x1, const double *x2, const double *v, const double *k,
                  const double *D, double *y, int ndim, const int64_t *dims, int circular,
                  const int64_t *lines, int64_t nlines, int nthreads) {
    geom g;
    if (!x1 || !x2 || !v || !k || !D || !y || make_geom(ndim, dims, &g)) return 1;
    job J;
    memset(&J, 0, sizeof J);
    if (circular < 0 || circular > 2) return 1;
    J.x1 = x1; J.x2 = x2; J.v = v; J.k = k; J.D = D; J.y = y; J.g = &g;
    J.circular = circular;
    J.items = lines;
    J.nitems = lines ? nlines : g.B * g.C;
    return run_jobs(&J, nthreads, direct_lines_worker);
}

/* out[i] = y at flat index idx[i] of the [B, C, L...] output tensor. */
int oracle_direct_points(const double *x1, const double *x2, const double *v, const double *k,
                         const double *D, int ndim, const int64_t *dims, int circular,
                         const int64_t *idx, int64_t npts, double *out, int nthreads) {
    geom g;
    if (!x1 || !x2 || !v || !k || !D || !idx || !out || make_geom(ndim, dims, &g)) return 1;
    for (int64_t i = 0; i < npts; ++i)
        if (idx[i] < 0 || idx[i] >= g.B * g.C * g.box) return 1;
    job J;
    memset(&J, 0, sizeof J);
    if (circular < 0 || circular > 2) return 1;
    J.x1 = x1; J.x2 = x2; J.v = v; J.k = k; J.D = D; J.y = out; J.g = &g;
    J.circular = circular;
    J.items = idx;
    J.nitems = npts;
    return run_jobs(&J, nthreads, direct_points_worker);
}

/* ------------------------------------------------------------------------- */
/* Convolution theorem with an own radix-2 FFT                                */
/* ------------------------------------------------------------------------- */

/* Table of exp(sign * 2 pi i j / n) for j < n/2 (n a power of two). */
static cplx *make_twiddles(int64_t n, int sign) {
    int64_t h = n / 2 > 0 ? n / 2 : 1;
    cplx *w = (cplx *)malloc((size_t)h * sizeof(cplx));
    if (!w) return NULL;
    for (int64_t j = 0; j < h; ++j) {
        double a = 2.0 * M_PI * (double)j / (double)n;
        w[j].re = cos(a);
        w[j].im = sign * sin(a);
    }
    return w;
}

/* In-place iterative radix-2 decimation-in-time FFT of a contiguous array:
 * X[f] = sum_n x[n] exp(sign 2 pi i f n / n_total), unnormalised.
 * tw = make_twiddles(n, sign). */
static void fft_radix2(cplx *a, int64_t n, const cplx *tw) {
    /* bit-reversal permutation */
    for (int64_t i = 1, j = 0; i < n; ++i) {
        int64_t bit = n >> 1;
        for (; j & bit; bit >>= 1) j ^= bit;
        j ^= bit;
        if (i < j) {
            cplx t = a[i];
            a[i] = a[j];
            a[j] = t;
        }
    }
    /* butterflies: blocks of length len, twiddle exp(sign 2 pi i j / len) */
    for (int64_t len = 2; len <= n; len <<= 1) {
        int64_t half = len >> 1, step = n / len;
        for (int64_t s = 0; s < n; s += len)
            for (int64_t j = 0; j < half; ++j) {
                cplx w = tw[j * step];
                cplx p = a[s + j], q = a[s + j + half];
                cplx t = {w.re * q.re - w.im * q.im, w.re * q.im + w.im * q.re};
                a[s + j].re = p.re + t.re;
                a[s + j].im = p.im + t.im;
                a[s + j + half].re = p.re - t.re;
                a[s + j + half].im = p.im - t.im;
            }
    }
}

static int is_pow2(int64_t n) { return n >= 1 && (n & (n - 1)) == 0; }

/* Exposed for pinning the FFT itself against a naive DFT.
 * data: interleaved (re, im) of length n; sign -1 forward, +1 inverse
 * (unnormalised either way). */
int oracle_fft1d(double *data, int64_t n, int sign) {
    if (!data || !is_pow2(n) || (sign != 1 && sign != -1)) return 1;
    cplx *tw = make_twiddles(n, sign);
    if (!tw) return 2;
    fft_radix2((cplx *)data, n, tw);
    free(tw);
    return 0;
}

/* FFT along axis `ax` of a 3-axis complex array with extents P[0..2]. */
static void fft_axis(cplx *a, const int64_t P[3], int ax, const cplx *tw, cplx *tmp) {
    int64_t n = P[ax];
    if (n == 1) return;
    int64_t stride = 1;
    for (int d = ax + 1; d < 3; ++d) stride *= P[d];
    int64_t outer = 1;
    for (int d = 0; d < ax; ++d) outer *= P[d];
    for (int64_t o = 0; o < outer; ++o)
        for (int64_t in = 0; in < stride; ++in) {
            cplx *base = a + o * n * stride + in;
            for (int64_t i = 0; i < n; ++i) tmp[i] = base[i * stride];
            fft_radix2(tmp, n, tw);
            for (int64_t i = 0; i < n; ++i) base[i * stride] = tmp[i];
        }
}

static void *fft_lines_worker(void *arg) {
    job *J = (job *)arg;
    const geom *g = J->g;
    int64_t P[3];
    int64_t tot = 1, maxP = 1;
    transform_extents(g, J->circular, P);
    for (int d = 0; d < 3; ++d) {
        tot *= P[d];
        if (P[d] > maxP) maxP = P[d];
    }
    cplx *U = (cplx *)malloc((size_t)tot * sizeof(cplx));
    cplx *K = (cplx *)malloc((size_t)tot * sizeof(cplx));
    cplx *tmp = (cplx *)malloc((size_t)maxP * sizeof(cplx));
    if (!U || !K || !tmp) {
        free(U); free(K); free(tmp);
        J->status = 2;
        return NULL;
    }
    const double scale = 1.0 / (double)tot;
    for (int64_t it = J->tid; it < J->nitems; it += J->nthreads) {
        int64_t line = item_at(J, it);
        int64_t base = line * g->box;
        int64_t c = line % g->C;
        /* 1. place u = x1*v and k on the padded grid, origin at index 0 */
        memset(U, 0, (size_t)tot * sizeof(cplx));
        memset(K, 0, (size_t)tot * sizeof(cplx));
        for (int64_t n0 = 0; n0 < g->L[0]; ++n0)
            for (int64_t n1 = 0; n1 < g->L[1]; ++n1)
                for (int64_t n2 = 0; n2 < g->L[2]; ++n2) {
                    int64_t src = base + (n0 * g->L[1] + n1) * g->L[2] + n2;
                    int64_t dst = (n0 * P[1] + n1) * P[2] + n2;
                    U[dst].re = J->x1[src] * J->v[src];
                    if (J->circular != MODE_CENTERED) K[dst].re = J->k[src];
                }
        if (J->circular == MODE_CENTERED) {
            /* displacement j_d - (L_d - 1) of kc goes to grid index
             * (j_d - (L_d - 1)) mod P_d */
            const int64_t K0 = 2 * g->L[0] - 1, K1 = 2 * g->L[1] - 1, K2 = 2 * g->L[2] - 1;
            const double *KC = J->k + line * centered_box(g);
            for (int64_t j0 = 0; j0 < K0; ++j0)
                for (int64_t j1 = 0; j1 < K1; ++j1)
                    for (int64_t j2 = 0; j2 < K2; ++j2) {
                        int64_t g0 = (j0 - (g->L[0] - 1) + P[0]) % P[0];
                        int64_t g1 = (j1 - (g->L[1] - 1) + P[1]) % P[1];
                        int64_t g2 = (j2 - (g->L[2] - 1) + P[2]) % P[2];
                        K[(g0 * P[1] + g1) * P[2] + g2].re = KC[(j0 * K1 + j1) * K2 + j2];
                    }
        }
        /* 2. forward transforms along every axis */
        for (int ax = 0; ax < 3; ++ax) {
            fft_axis(U, P, ax, J->tw_fwd[ax], tmp);
            fft_axis(K, P, ax, J->tw_fwd[ax], tmp);
        }
        /* 3. pointwise product of the spectra */
        for (int64_t i = 0; i < tot; ++i) {
            cplx a = U[i], b = K[i];
            U[i].re = a.re * b.re - a.im * b.im;
            U[i].im = a.re * b.im + a.im * b.re;
        }
        /* 4. inverse along every axis, scaled by 1/prod(P) */
        for (int ax = 0; ax < 3; ++ax) fft_axis(U, P, ax, J->tw_inv[ax], tmp);
        /* 5. crop to [0, L), check the result is real, add skip, gate */
        double maxre = 0.0, maxim = 0.0;
        for (int64_t n0 = 0; n0 < g->L[0]; ++n0)
            for (int64_t n1 = 0; n1 < g->L[1]; ++n1)
                for (int64_t n2 = 0; n2 < g->L[2]; ++n2) {
                    int64_t src = base + (n0 * g->L[1] + n1) * g->L[2] + n2;
                    int64_t pos = (n0 * P[1] + n1) * P[2] + n2;
                    double conv = U[pos].re * scale;
                    double im = fabs(U[pos].im * scale);
                    if (fabs(conv) > maxre) maxre = fabs(conv);
                    if (im > maxim) maxim = im;
                    double u = J->x1[src] * J->v[src];
                    J->y[src] = J->x2[src] * (conv + J->D[c] * u);
                }
        if (maxim > 1e-9 * (maxre > 1e-300 ? maxre : 1e-300) && maxim > 1e-200) J->status = 3;
    }
    free(U);
    free(K);
    free(tmp);
    return NULL;
}

int oracle_fft(const double *x1, const double *x2, const double *v, const double *k,
               const double *D, double *y, int ndim, const int64_t *dims, int circular,
               const int64_t *lines, int64_t nlines, int nthreads) {
    geom g;
    if (!x1 || !x2 || !v || !k || !D || !y || make_geom(ndim, dims, &g)) return 1;
    if (circular < 0 || circular > 2) return 1;
    if (circular == MODE_CIRCULAR)
        for (int d = 0; d < 3; ++d)
            if (!is_pow2(g.L[d])) return 1;
    int64_t P[3];
    transform_extents(&g, circular == MODE_CIRCULAR ? MODE_CIRCULAR : MODE_LINEAR, P);
    cplx *twf[3] = {NULL, NULL, NULL}, *twi[3] = {NULL, NULL, NULL};
    int rc = 0;
    for (int d = 0; d < 3; ++d) {
        twf[d] = make_twiddles(P[d], -1);
        twi[d] = make_twiddles(P[d], +1);
        if (!twf[d] || !twi[d]) rc = 2;
    }
    if (!rc) {
        job J;
        memset(&J, 0, sizeof J);
        J.x1 = x1; J.x2 = x2; J.v = v; J.k = k; J.D = D; J.y = y; J.g = &g;
        J.circular = circular;
        J.items = lines;
        J.nitems = lines ? nlines : g.B * g.C;
        J.tw_fwd = (const cplx *const *)twf;
        J.tw_inv = (const cplx *const *)twi;
        rc = run_jobs(&J, nthreads, fft_lines_worker);
    }
    for (int d = 0; d < 3; ++d) {
        free(twf[d]);
        free(twi[d]);
    }
    return rc;
}

/* ------------------------------------------------------------------------- */
/* Backward                                                                   */
/* ------------------------------------------------------------------------- */

typedef struct {
    const double *x1, *x2, *v, *k, *D, *gy;
    double *gx1, *gx2, *gv, *gk, *hu; /* hu: per-line sum of h u */
    const geom *g;
    int circular;
    int tid, nthreads;
    int status;
    const cplx *const *tw_fwd;
    const cplx *const *tw_inv;
} bjob;

static void unflat(const geom *g, int64_t r, int64_t n[3]) {
    n[2] = r % g->L[2];
    n[1] = (r / g->L[2]) % g->L[1];
    n[0] = r / (g->L[2] * g->L[1]);
}

/* Index of a - b on the grid: linear requires a_d >= b_d (else -1);
 * circular wraps each axis. */
static int64_t diff_index(const geom *g, const int64_t a[3], const int64_t b[3], int circular) {
    int64_t r = 0;
    for (int d = 0; d < 3; ++d) {
        int64_t x = a[d] - b[d];
        if (circular)
            x = (x % g->L[d] + g->L[d]) % g->L[d];
        else if (x < 0)
            return -1;
        r = r * g->L[d] + x;
    }
    return r;
}

static void *backward_direct_worker(void *arg) {
    bjob *J = (bjob *)arg;
    const geom *g = J->g;
    const int64_t box = g->box;
    double *u = (double *)malloc((size_t)box * sizeof(double));
    double *h = (double *)malloc((size_t)box * sizeof(double));
    if (!u || !h) {
        free(u); free(h);
        J->status = 2;
        return NULL;
    }
    for (int64_t line = J->tid; line < g->B * g->C; line += J->nthreads) {
        const int64_t base = line * box, c = line % g->C;
        const double *K = J->k + base;
        for (int64_t i = 0; i < box; ++i) {
            u[i] = J->x1[base + i] * J->v[base + i];
            h[i] = J->gy[base + i] * J->x2[base + i];
        }
        double hu = 0.0;
        for (int64_t i = 0; i < box; ++i) hu += h[i] * u[i];
        J->hu[line] = hu;
        for (int64_t i = 0; i < box; ++i) {
            int64_t p[3], q[3];
            unflat(g, i, p);
            /* z[i] = sum_m k[m] u[i - m] + D u[i] */
            double conv = 0.0, gu = 0.0, gk = 0.0;
            for (int64_t m = 0; m < box; ++m) {
                unflat(g, m, q);
                int64_t im = diff_index(g, p, q, J->circular); /* i - m */
                if (im >= 0) conv += K[m] * u[im];
            }
            /* gu[i] = sum_n k[n - i] h[n];  gk[i] = sum_n h[n] u[n - i] */
            for (int64_t n = 0; n < box; ++n) {
                unflat(g, n, q);
                int64_t ni = diff_index(g, q, p, J->circular); /* n - i */
                if (ni >= 0) {
                    gu += K[ni] * h[n];
                    gk += h[n] * u[ni];
                }
            }
            const double z = conv + J->D[c] * u[i];
            J->gx2[base + i] = J->gy[base + i] * z;
            gu += J->D[c] * h[i];
            J->gx1[base + i] = gu * J->v[base + i];
            J->gv[base + i] = gu * J->x1[base + i];
            J->gk[base + i] = gk;
        }
    }
    free(u);
    free(h);
    return NULL;
}

/* centred mode: conv[n] = sum_m kc[n - m + (L - 1)] u[m], kc on the 2 L_d - 1
 * point grid, so gu[j] = sum_n kc[n - j + (L - 1)] h[n] + D h[j] and
 * gk[i] = sum_n h[n] u[n - i + (L - 1)] (where that index is on the grid) */
static int64_t kc_index(const geom *g, const int64_t a[3], const int64_t b[3]) {
    int64_t r = 0;
    for (int d = 0; d < 3; ++d) r = r * (2 * g->L[d] - 1) + (a[d] - b[d] + g->L[d] - 1);
    return r;
}

static void *backward_centered_worker(void *arg) {
    bjob *J = (bjob *)arg;
    const geom *g = J->g;
    const int64_t box = g->box, kbox = centered_box(g);
    double *u = (double *)malloc((size_t)box * sizeof(double));
    double *h = (double *)malloc((size_t)box * sizeof(double));
    if (!u || !h) {
        free(u); free(h);
        J->status = 2;
        return NULL;
    }
    for (int64_t line = J->tid; line < g->B * g->C; line += J->nthreads) {
        const int64_t base = line * box, kbase = line * kbox, c = line % g->C;
        const double *K = J->k + kbase;
        double hu = 0.0;
        for (int64_t i = 0; i < box; ++i) {
            u[i] = J->x1[base + i] * J->v[base + i];
            h[i] = J->gy[base + i] * J->x2[base + i];
            hu += h[i] * u[i];
        }
        J->hu[line] = hu;
        for (int64_t i = 0; i < box; ++i) {
            int64_t p[3], q[3];
            unflat(g, i, p);
            double conv = 0.0, gu = 0.0;
            for (int64_t m = 0; m < box; ++m) {
                unflat(g, m, q);
                conv += K[kc_index(g, p, q)] * u[m];  /* kc[i - m + L - 1] u[m] */
                gu += K[kc_index(g, q, p)] * h[m];    /* kc[m - i + L - 1] h[m] */
            }
            const double z = conv + J->D[c] * u[i];
            J->gx2[base + i] = J->gy[base + i] * z;
            gu += J->D[c] * h[i];
            J->gx1[base + i] = gu * J->v[base + i];
            J->gv[base + i] = gu * J->x1[base + i];
        }
        for (int64_t ki = 0; ki < kbox; ++ki) {
            /* kernel point ki: displacement e_d = index_d - (L_d - 1) */
            int64_t e[3], r = ki;
            for (int d = 2; d >= 0; --d) {
                e[d] = r % (2 * g->L[d] - 1) - (g->L[d] - 1);
                r /= 2 * g->L[d] - 1;
            }
            double s = 0.0;
            for (int64_t n = 0; n < box; ++n) {
                int64_t q[3], m = 0, ok = 1;
                unflat(g, n, q);
                for (int d = 0; d < 3; ++d) {
                    const int64_t x = q[d] - e[d];
                    if (x < 0 || x >= g->L[d]) ok = 0;
                    m = m * g->L[d] + x;
                }
                if (ok) s += h[n] * u[m];
            }
            J->gk[kbase + ki] = s;
        }
    }
    free(u);
    free(h);
    return NULL;
}

static void *backward_fft_worker(void *arg) {
    bjob *J = (bjob *)arg;
    const geom *g = J->g;
    int64_t P[3];
    int64_t tot = 1, maxP = 1;
    transform_extents(g, J->circular, P);
    for (int d = 0; d < 3; ++d) {
        tot *= P[d];
        if (P[d] > maxP) maxP = P[d];
    }
    cplx *U = (cplx *)malloc((size_t)tot * sizeof(cplx));
    cplx *K = (cplx *)malloc((size_t)tot * sizeof(cplx));
    cplx *H = (cplx *)malloc((size_t)tot * sizeof(cplx));
    cplx *Z = (cplx *)malloc((size_t)tot * sizeof(cplx));
    cplx *tmp = (cplx *)malloc((size_t)maxP * sizeof(cplx));
    if (!U || !K || !H || !Z || !tmp) {
        free(U); free(K); free(H); free(Z); free(tmp);
        J->status = 2;
        return NULL;
    }
    const double scale = 1.0 / (double)tot;
    for (int64_t line = J->tid; line < g->B * g->C; line += J->nthreads) {
        const int64_t base = line * g->box, c = line % g->C;
        memset(U, 0, (size_t)tot * sizeof(cplx));
        memset(K, 0, (size_t)tot * sizeof(cplx));
        memset(H, 0, (size_t)tot * sizeof(cplx));
        double hu = 0.0;
        for (int64_t n0 = 0; n0 < g->L[0]; ++n0)
            for (int64_t n1 = 0; n1 < g->L[1]; ++n1)
                for (int64_t n2 = 0; n2 < g->L[2]; ++n2) {
                    int64_t src = base + (n0 * g->L[1] + n1) * g->L[2] + n2;
                    int64_t dst = (n0 * P[1] + n1) * P[2] + n2;
                    U[dst].re = J->x1[src] * J->v[src];
                    K[dst].re = J->k[src];
                    H[dst].re = J->gy[src] * J->x2[src];
                    hu += H[dst].re * U[dst].re;
                }
        J->hu[line] = hu;
        for (int ax = 0; ax < 3; ++ax) {
            fft_axis(U, P, ax, J->tw_fwd[ax], tmp);
            fft_axis(K, P, ax, J->tw_fwd[ax], tmp);
            fft_axis(H, P, ax, J->tw_fwd[ax], tmp);
        }
        /* Z = U K, then H <- conj(K) H (for gu) and K <- conj(U) H (for gk) */
        for (int64_t i = 0; i < tot; ++i) {
            cplx a = U[i], b = K[i], e = H[i];
            Z[i].re = a.re * b.re - a.im * b.im;
            Z[i].im = a.re * b.im + a.im * b.re;
            H[i].re = b.re * e.re + b.im * e.im;
            H[i].im = b.re * e.im - b.im * e.re;
            K[i].re = a.re * e.re + a.im * e.im;
            K[i].im = a.re * e.im - a.im * e.re;
        }
        for (int ax = 0; ax < 3; ++ax) {
            fft_axis(Z, P, ax, J->tw_inv[ax], tmp);
            fft_axis(H, P, ax, J->tw_inv[ax], tmp);
            fft_axis(K, P, ax, J->tw_inv[ax], tmp);
        }
        double maxre = 0.0, maxim = 0.0;
        for (int64_t n0 = 0; n0 < g->L[0]; ++n0)
            for (int64_t n1 = 0; n1 < g->L[1]; ++n1)
                for (int64_t n2 = 0; n2 < g->L[2]; ++n2) {
                    int64_t src = base + (n0 * g->L[1] + n1) * g->L[2] + n2;
                    int64_t pos = (n0 * P[1] + n1) * P[2] + n2;
                    const cplx *outs[3] = {&Z[pos], &H[pos], &K[pos]};
                    for (int o = 0; o < 3; ++o) {
                        double re = fabs(outs[o]->re * scale), im = fabs(outs[o]->im * scale);
                        if (re > maxre) maxre = re;
                        if (im > maxim) maxim = im;
                    }
                    const double u = J->x1[src] * J->v[src];
                    const double hh = J->gy[src] * J->x2[src];
                    const double z = Z[pos].re * scale + J->D[c] * u;
                    const double gu = H[pos].re * scale + J->D[c] * hh;
                    J->gx2[src] = J->gy[src] * z;
                    J->gx1[src] = gu * J->v[src];
                    J->gv[src] = gu * J->x1[src];
                    J->gk[src] = K[pos].re * scale;
                }
        if (maxim > 1e-9 * (maxre > 1e-300 ? maxre : 1e-300) && maxim > 1e-200) J->status = 3;
    }
    free(U); free(K); free(H); free(Z); free(tmp);
    return NULL;
}

static int run_bjobs(bjob *proto, int nthreads, void *(*fn)(void *)) {
    if (nthreads < 1) nthreads = 1;
    if (nthreads > 256) nthreads = 256;
    bjob jobs[256];
    pthread_t th[256];
    int started[256];
    int rc = 0;
    for (int t = 0; t < nthreads; ++t) {
        jobs[t] = *proto;
        jobs[t].tid = t;
        jobs[t].nthreads = nthreads;
        jobs[t].status = 0;
        started[t] = 0;
    }
    for (int t = 1; t < nthreads; ++t) {
        if (pthread_create(&th[t], NULL, fn, &jobs[t]) == 0)
            started[t] = 1;
        else
            rc = 4;
    }
    fn(&jobs[0]);
    for (int t = 1; t < nthreads; ++t)
        if (started[t]) pthread_join(th[t], NULL);
    if (rc) return rc;
    for (int t = 0; t < nthreads; ++t)
        if (jobs[t].status) return jobs[t].status;
    return 0;
}

static int backward_common(const double *x1, const double *x2, const double *v, const double *k,
                           const double *D, const double *gy, double *gx1, double *gx2, double *gv,
                           double *gk, double *gD, int ndim, const int64_t *dims, int circular,
                           int nthreads, int use_fft) {
    geom g;
    if (!x1 || !x2 || !v || !k || !D || !gy || !gx1 || !gx2 || !gv || !gk || !gD ||
        make_geom(ndim, dims, &g))
        return 1;
    if (circular != MODE_LINEAR && circular != MODE_CIRCULAR && circular != MODE_CENTERED) return 1;
    if (use_fft && circular == MODE_CENTERED) return 1; /* the centred backward is the direct sums */
    if (use_fft && circular == MODE_CIRCULAR)
        for (int d = 0; d < 3; ++d)
            if (!is_pow2(g.L[d])) return 1;
    double *hu = (double *)calloc((size_t)(g.B * g.C), sizeof(double));
    if (!hu) return 2;
    int64_t P[3];
    transform_extents(&g, circular == MODE_CIRCULAR ? MODE_CIRCULAR : MODE_LINEAR, P);
    cplx *twf[3] = {NULL, NULL, NULL}, *twi[3] = {NULL, NULL, NULL};
    int rc = 0;
    if (use_fft)
        for (int d = 0; d < 3; ++d) {
            twf[d] = make_twiddles(P[d], -1);
            twi[d] = make_twiddles(P[d], +1);
            if (!twf[d] || !twi[d]) rc = 2;
        }
    if (!rc) {
        bjob J;
        memset(&J, 0, sizeof J);
        J.x1 = x1; J.x2 = x2; J.v = v; J.k = k; J.D = D; J.gy = gy;
        J.gx1 = gx1; J.gx2 = gx2; J.gv = gv; J.gk = gk; J.hu = hu; J.g = &g;
        J.circular = circular == MODE_CIRCULAR ? 1 : 0;
        J.tw_fwd = (const cplx *const *)twf;
        J.tw_inv = (const cplx *const *)twi;
        rc = run_bjobs(&J, nthreads,
                       use_fft ? backward_fft_worker
                               : (circular == MODE_CENTERED ? backward_centered_worker : backward_direct_worker));
    }
    if (!rc) /* gD[c] = sum over samples, in sample order */
        for (int64_t c = 0; c < g.C; ++c) {
            double s = 0.0;
            for (int64_t b = 0; b < g.B; ++b) s += hu[b * g.C + c];
            gD[c] = s;
        }
    for (int d = 0; d < 3; ++d) {
        free(twf[d]);
        free(twi[d]);
    }
    free(hu);
    return rc;
}

int oracle_backward_direct(const double *x1, const double *x2, const double *v, const double *k,
                           const double *D, const double *gy, double *gx1, double *gx2, double *gv,
                           double *gk, double *gD, int ndim, const int64_t *dims, int circular,
                           int nthreads) {
    return backward_common(x1, x2, v, k, D, gy, gx1, gx2, gv, gk, gD, ndim, dims, circular, nthreads, 0);
}

int oracle_backward_fft(const double *x1, const double *x2, const double *v, const double *k,
                        const double *D, const double *gy, double *gx1, double *gx2, double *gv,
                        double *gk, double *gD, int ndim, const int64_t *dims, int circular,
                        int nthreads) {
    return backward_common(x1, x2, v, k, D, gy, gx1, gx2, gv, gk, gD, ndim, dims, circular, nthreads, 1);
}

int oracle_version(void) { return 7; }

/* ------------------------------------------------------------------------- */
/* HyenaND operator: normalised prologue, long convolution, normalised       */
/* epilogue                                                                  */
/* ------------------------------------------------------------------------- */

static double silu(double x) { return x / (1.0 + exp(-x)); }
static double sigmoid(double x) { return 1.0 / (1.0 + exp(-x)); }

int oracle_operator(const double *q, const double *kin, const double *vin, const double *k,
                    const double *D, const double *w_in, const double *w_out, double eps_l2,
                    double eps_rms, double *y, int ndim, const int64_t *dims, int mode,
                    int nthreads) {
    geom g;
    if (!q || !kin || !vin || !k || !D || !w_in || !w_out || !y || make_geom(ndim, dims, &g)) return 1;
    if (mode < 0 || mode > 2 || !(eps_l2 >= 0.0) || !(eps_rms >= 0.0)) return 1;
    const int64_t B = g.B, C = g.C, box = g.box, n = B * C * box;
    double *u = (double *)malloc((size_t)n * sizeof(double));
    double *gate = (double *)malloc((size_t)n * sizeof(double));
    double *ones = (double *)malloc((size_t)n * sizeof(double));
    if (!u || !gate || !ones) {
        free(u); free(gate); free(ones);
        return 2;
    }
    /* 1. prologue, one channel vector per (b, p) */
    for (int64_t b = 0; b < B; ++b)
        for (int64_t p = 0; p < box; ++p) {
            double qq = 0.0;
            for (int64_t c = 0; c < C; ++c) {
                double x = q[(b * C + c) * box + p];
                qq += x * x;
            }
            double qn = sqrt(qq);
            if (qn < eps_l2) qn = eps_l2;
            double aa = 0.0;
            for (int64_t c = 0; c < C; ++c) {
                int64_t i = (b * C + c) * box + p;
                double a = (qn > 0.0 ? q[i] / qn : 0.0) * silu(kin[i]);
                u[i] = a;
                aa += a * a;
            }
            double r = sqrt(aa / (double)C + eps_rms);
            for (int64_t c = 0; c < C; ++c) {
                int64_t i = (b * C + c) * box + p;
                u[i] = (r > 0.0 ? u[i] / r : 0.0) * w_in[c];
            }
        }
    for (int64_t i = 0; i < n; ++i) {
        gate[i] = sigmoid(vin[i]);
        ones[i] = 1.0;
    }
    /* 2. the gated long convolution of u (x1 = u, v = 1, x2 = the gate);
       the circular mode on extents that are not powers of two takes the
       direct sums (this file's FFT is radix 2) */
    int pow2_grid = 1;
    for (int d = 0; d < 3; ++d) pow2_grid = pow2_grid && is_pow2(g.L[d]);
    int rc = (mode == MODE_CIRCULAR && !pow2_grid)
                 ? oracle_direct(u, gate, ones, k, D, y, ndim, dims, mode, NULL, 0, nthreads)
                 : oracle_fft(u, gate, ones, k, D, y, ndim, dims, mode, NULL, 0, nthreads);
    /* 3. epilogue RMSNorm across channels */
    if (!rc)
        for (int64_t b = 0; b < B; ++b)
            for (int64_t p = 0; p < box; ++p) {
                double zz = 0.0;
                for (int64_t c = 0; c < C; ++c) {
                    double z = y[(b * C + c) * box + p];
                    zz += z * z;
                }
                double r = sqrt(zz / (double)C + eps_rms);
                for (int64_t c = 0; c < C; ++c) {
                    int64_t i = (b * C + c) * box + p;
                    y[i] = (r > 0.0 ? y[i] / r : 0.0) * w_out[c];
                }
            }
    free(u);
    free(gate);
    free(ones);
    return rc;
}

/* ------------------------------------------------------------------------- */
/* Kernel synthesis: the implicit, input-dependent kernel K(x)               */
/* ------------------------------------------------------------------------- */
/*
 * oracle_kernel_synth -- the HyenaND kernel evaluated on the kernel grid of a
 * convolution (section 3.2.1 "Multi-Dimensional Continuous Convolutional
 * Kernels", Eq. (kernel); section 3.2.2 "Input-Dependent Kernels via
 * Registers and FiLM", Eq. (film); the appendix "HyenaND Design Details:
 * Masking and Initialization", Eq. (mask)):
 *
 *   h_1 = sin(omega0 * (r W1) + b_1)          r in [-1, 1]^N, W1 [N, Hf]
 *   h_j = sin(h_{j-1} W_j + b_j)              j = 2 .. J, W_j [Hf, Hf]
 *   after each sine: h_j <- gamma_j[b] * h_j + beta_j[b]   (FiLM, per sample)
 *   f   = h_J Wout                            Wout [Hf, C]
 *   K[b, c, i] = w_c(r_i) f[c]
 *
 * Window w_c: kind 0, the Gaussian of Eq. (mask), exp(-1/2 sum_d (r_d /
 * sigma[d, c])^2) with win = sigma [N, C]; kind 1, the exponential decay
 * exp(-alpha[c] sum_d |r_d|) of the original Hyena window (one axis: Hyena's
 * exp(-alpha |r|)) with win = alpha [C].
 *
 * The grid follows the convolution's kernel layout: per axis L_d points in
 * the linear and circular modes, 2 L_d - 1 in the centered mode.  The point's
 * displacement is i (linear), i - (L_d - 1) (centered), i for i <= L_d / 2
 * and i - L_d beyond (circular, the signed periodic displacement), and its
 * coordinate r_d = displacement / (L_d - 1) (0 when L_d = 1): the double
 * grid of the centered mode spans [-1, 1] exactly, and every mode gives one
 * displacement the same coordinate.
 *
 * Readings: the hidden-layer frequency of the appendix's SIREN definition is
 * taken as folded into W_j; the bias is that definition's (one per layer, may
 * be NULL for none); FiLM acts on the sine's output, the hidden activation.
 * gamma and beta are [B, J, Hf]; both NULL gives the unmodulated kernel of
 * section 3.2.1, written once as [C, grid] (a kernel shared by the batch).
 * Wh is [J - 1, Hf, Hf], row = input unit.  k is [B, C, grid] or [C, grid].
 */
static double synth_coord(int64_t i, int64_t L, int mode) {
    if (L <= 1) return 0.0;
    int64_t d;
    if (mode == MODE_CENTERED)
        d = i - (L - 1);
    else if (mode == MODE_CIRCULAR)
        d = i <= L / 2 ? i : i - L;
    else
        d = i;
    return (double)d / (double)(L - 1);
}

int oracle_kernel_synth(const double *omega0, const double *W1, const double *Wh, const double *bias,
                        const double *gamma, const double *beta, const double *Wout, const double *win,
                        int wkind, double *k, int ndim, const int64_t *dims, int mode, int hidden,
                        int layers) {
    geom g;
    if (!omega0 || !W1 || !Wout || !win || !k || make_geom(ndim, dims, &g)) return 1;
    if (mode < 0 || mode > 2 || wkind < 0 || wkind > 1 || hidden < 1 || layers < 1) return 1;
    if ((gamma == NULL) != (beta == NULL) || (layers > 1 && !Wh)) return 1;
    const int64_t C = g.C, H = hidden, J = layers;
    const int64_t nb = gamma ? g.B : 1;
    int64_t KL[3];
    for (int d = 0; d < 3; ++d) KL[d] = (mode == MODE_CENTERED) ? 2 * g.L[d] - 1 : g.L[d];
    const int64_t npos = KL[0] * KL[1] * KL[2];
    double *h = (double *)malloc((size_t)H * sizeof(double));
    double *t = (double *)malloc((size_t)H * sizeof(double));
    if (!h || !t) {
        free(h);
        free(t);
        return 2;
    }
    for (int64_t b = 0; b < nb; ++b)
        for (int64_t p = 0; p < npos; ++p) {
            /* coordinates of the grid point; axis a of the N real axes is
               axis 3 - N + a of the padded three */
            int64_t idx[3] = {p / (KL[1] * KL[2]), (p / KL[2]) % KL[1], p % KL[2]};
            double r[3];
            for (int a = 0; a < ndim; ++a) {
                int d = 3 - ndim + a;
                r[a] = synth_coord(idx[d], g.L[d], mode);
            }
            /* first layer */
            for (int64_t o = 0; o < H; ++o) {
                double s = 0.0;
                for (int a = 0; a < ndim; ++a) s += r[a] * W1[a * H + o];
                s = omega0[o] * s + (bias ? bias[o] : 0.0);
                h[o] = sin(s);
                if (gamma) h[o] = gamma[(b * J + 0) * H + o] * h[o] + beta[(b * J + 0) * H + o];
            }
            /* hidden layers 2 .. J */
            for (int64_t j = 1; j < J; ++j) {
                const double *W = Wh + (j - 1) * H * H;
                for (int64_t o = 0; o < H; ++o) {
                    double s = 0.0;
                    for (int64_t i = 0; i < H; ++i) s += h[i] * W[i * H + o];
                    s += bias ? bias[j * H + o] : 0.0;
                    t[o] = sin(s);
                    if (gamma) t[o] = gamma[(b * J + j) * H + o] * t[o] + beta[(b * J + j) * H + o];
                }
                memcpy(h, t, (size_t)H * sizeof(double));
            }
            /* output projection and window */
            for (int64_t c = 0; c < C; ++c) {
                double f = 0.0;
                for (int64_t i = 0; i < H; ++i) f += h[i] * Wout[i * C + c];
                double w;
                if (wkind == 0) {
                    double e = 0.0;
                    for (int a = 0; a < ndim; ++a) {
                        double z = r[a] / win[a * C + c];
                        e += z * z;
                    }
                    w = exp(-0.5 * e);
                } else {
                    double e = 0.0;
                    for (int a = 0; a < ndim; ++a) e += fabs(r[a]);
                    w = exp(-win[c] * e);
                }
                k[(b * C + c) * npos + p] = w * f;
            }
        }
    free(h);
    free(t);
    return 0;
}

/* ------------------------------------------------------------------------- */
/* Modal filter generation                                                   */
/* ------------------------------------------------------------------------- */
/*
 * oracle_modal_filter -- the implicit modal filter of order M of the long
 * convolution layers (appendix "Filter Generation"): per channel c a sum of
 * M damped complex exponentials, taken as its real part,
 *
 *   k[c, t] = Re sum_m R[c, m] lambda[c, m]^t,   t = 0 .. L - 1,
 *   lambda = exp(a + i theta),  R = re + i im,
 *
 * so k[c, t] = sum_m exp(t a) (re cos(t theta) - im sin(t theta)).  The
 * paper gives the order (16) and the form only by name; this is the modal
 * (sum of poles and residues) form with the pole given by its log-magnitude
 * a and angle theta.  a, theta, re, im are [C, M]; k is [C, L].  t * theta
 * is formed in double, which holds the product of an fp32 angle and t < 2^29
 * exactly.
 */
int oracle_modal_filter(const double *a, const double *theta, const double *re, const double *im, double *k,
                        int64_t C, int64_t M, int64_t L) {
    if (!a || !theta || !re || !im || !k || C < 1 || M < 1 || L < 1) return 1;
    for (int64_t c = 0; c < C; ++c)
        for (int64_t t = 0; t < L; ++t) {
            double s = 0.0;
            for (int64_t m = 0; m < M; ++m) {
                const int64_t i = c * M + m;
                const double ph = (double)t * theta[i];
                s += exp((double)t * a[i]) * (re[i] * cos(ph) - im[i] * sin(ph));
            }
            k[c * L + t] = s;
        }
    return 0;
}
