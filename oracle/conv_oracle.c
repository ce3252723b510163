/*
 * fp64 reference convolutions — TEST INFRASTRUCTURE ONLY.
 *
 * This file is the oracle that the HIP library is checked against. It is
 * deliberately slow and plain: every output element is computed on its own
 * from the definition of the operation, with a sequential fp64 sum over the
 * terms in a fixed order. It shares no code, header, table or index helper
 * with the GPU library, and nothing in the product path may link or call it.
 *
 * Operations (all tensors are fp64 here; the caller upcasts fp16 exactly):
 *   fwd        y[n,p,q,k]  = sum_{r,s,c} x~[n, p*sh-ph+r, q*sw-pw+s, c] * W[k,r,s,c]
 *   bwd_data   dx[n,h,w,c] = sum over (k,r,s) such that (h+ph-r) is a multiple
 *                            of sh with quotient p in [0,P), same for w with q,
 *                            of dy[n,p,q,k] * W[k,r,s,c]
 *   bwd_weight dW[k,r,s,c] = sum_{n,p,q} dy[n,p,q,k] * x~[n, p*sh-ph+r, q*sw-pw+s, c]
 *   convT fwd  y[n,o,u,k]  = sum over (c,r,s) such that (o+ph-r) is a multiple
 *                            of sh with quotient i in [0,H), same for u with j,
 *                            of x[n,i,j,c] * Wt[c,r,s,k]
 * where x~ is x extended by zeros outside the image. The number of the
 * multiply-adds is the direct-convolution operation count of the paper
 * (Section 5.2, equation OPS_conv); the three training passes (forward,
 * kernel gradient, input gradient) are the three operations whose sum the
 * paper's performance definitions count (Section 5.2, the factor of 3).
 * Layouts: activations NHWC, conv weights KRSC, transposed-conv weights
 * C_in x R x S x C_out. Convolution is cross-correlation (no kernel flip).
 * Output size of fwd: P = floor((H + 2*ph - R)/sh) + 1; of convT:
 * Ho = (H - 1)*sh - 2*ph + R.
 *
 * Each op has an element function (one output, from the formula), a full
 * version (every output, OpenMP over output elements) and a sampled version
 * (a caller-given list of flat output indices).
 */
#include <stdint.h>

typedef struct {
    int64_t n, h, w, c;     /* input image of the forward conv (convT: its input) */
    int64_t k, r, s;        /* output channels, kernel height, kernel width       */
    int64_t sh, sw, ph, pw; /* stride and padding                                 */
} ocs;

static int64_t fwd_out(int64_t in, int64_t pad, int64_t ker, int64_t str) {
    return (in + 2 * pad - ker) / str + 1;
}

static int64_t convt_out(int64_t in, int64_t pad, int64_t ker, int64_t str) {
    return (in - 1) * str - 2 * pad + ker;
}

/* ---- forward ---------------------------------------------------------- */
static double fwd_elem(const ocs *g, const double *x, const double *W,
                       int64_t n, int64_t p, int64_t q, int64_t k) {
    double acc = 0.0;
    for (int64_t r = 0; r < g->r; ++r) {
        int64_t hi = p * g->sh - g->ph + r;
        if (hi < 0 || hi >= g->h) continue;
        for (int64_t s = 0; s < g->s; ++s) {
            int64_t wi = q * g->sw - g->pw + s;
            if (wi < 0 || wi >= g->w) continue;
            const double *xp = x + ((n * g->h + hi) * g->w + wi) * g->c;
            const double *wp = W + ((k * g->r + r) * g->s + s) * g->c;
            for (int64_t c = 0; c < g->c; ++c) acc += xp[c] * wp[c];
        }
    }
    return acc;
}

/* ---- backward data (adjoint of fwd w.r.t. x) -------------------------- */
static double bwd_data_elem(const ocs *g, const double *dy, const double *W,
                            int64_t n, int64_t h, int64_t w, int64_t c) {
    int64_t P = fwd_out(g->h, g->ph, g->r, g->sh);
    int64_t Q = fwd_out(g->w, g->pw, g->s, g->sw);
    double acc = 0.0;
    for (int64_t r = 0; r < g->r; ++r) {
        int64_t t = h + g->ph - r;
        if (t < 0 || t % g->sh != 0) continue;
        int64_t p = t / g->sh;
        if (p >= P) continue;
        for (int64_t s = 0; s < g->s; ++s) {
            int64_t u = w + g->pw - s;
            if (u < 0 || u % g->sw != 0) continue;
            int64_t q = u / g->sw;
            if (q >= Q) continue;
            const double *dyp = dy + ((n * P + p) * Q + q) * g->k;
            for (int64_t k = 0; k < g->k; ++k)
                acc += dyp[k] * W[((k * g->r + r) * g->s + s) * g->c + c];
        }
    }
    return acc;
}

/* ---- backward weight (gradient of <fwd(x;W), dy> w.r.t. W) ------------ */
static double bwd_weight_elem(const ocs *g, const double *x, const double *dy,
                              int64_t k, int64_t r, int64_t s, int64_t c) {
    int64_t P = fwd_out(g->h, g->ph, g->r, g->sh);
    int64_t Q = fwd_out(g->w, g->pw, g->s, g->sw);
    double acc = 0.0;
    for (int64_t n = 0; n < g->n; ++n)
        for (int64_t p = 0; p < P; ++p) {
            int64_t hi = p * g->sh - g->ph + r;
            if (hi < 0 || hi >= g->h) continue;
            for (int64_t q = 0; q < Q; ++q) {
                int64_t wi = q * g->sw - g->pw + s;
                if (wi < 0 || wi >= g->w) continue;
                acc += dy[((n * P + p) * Q + q) * g->k + k] *
                       x[((n * g->h + hi) * g->w + wi) * g->c + c];
            }
        }
    return acc;
}

/* ---- transposed-conv forward (scatter form, evaluated per output) ----- */
static double convt_elem(const ocs *g, const double *x, const double *Wt,
                         int64_t n, int64_t o, int64_t u, int64_t k) {
    double acc = 0.0;
    for (int64_t r = 0; r < g->r; ++r) {
        int64_t t = o + g->ph - r;
        if (t < 0 || t % g->sh != 0) continue;
        int64_t i = t / g->sh;
        if (i >= g->h) continue;
        for (int64_t s = 0; s < g->s; ++s) {
            int64_t v = u + g->pw - s;
            if (v < 0 || v % g->sw != 0) continue;
            int64_t j = v / g->sw;
            if (j >= g->w) continue;
            const double *xp = x + ((n * g->h + i) * g->w + j) * g->c;
            for (int64_t c = 0; c < g->c; ++c)
                acc += xp[c] * Wt[((c * g->r + r) * g->s + s) * g->k + k];
        }
    }
    return acc;
}

/* ---- drivers ---------------------------------------------------------- */
enum { OP_FWD = 0, OP_BWD_DATA = 1, OP_BWD_WEIGHT = 2, OP_CONVT = 3 };

/* Output dims (d0,d1,d2,d3) of op in row-major order. */
static void out_dims(const ocs *g, int op, int64_t d[4]) {
    switch (op) {
    case OP_FWD:
        d[0] = g->n; d[1] = fwd_out(g->h, g->ph, g->r, g->sh);
        d[2] = fwd_out(g->w, g->pw, g->s, g->sw); d[3] = g->k; break;
    case OP_BWD_DATA:
        d[0] = g->n; d[1] = g->h; d[2] = g->w; d[3] = g->c; break;
    case OP_BWD_WEIGHT:
        d[0] = g->k; d[1] = g->r; d[2] = g->s; d[3] = g->c; break;
    default:
        d[0] = g->n; d[1] = convt_out(g->h, g->ph, g->r, g->sh);
        d[2] = convt_out(g->w, g->pw, g->s, g->sw); d[3] = g->k; break;
    }
}

static double elem(const ocs *g, int op, const double *a, const double *b,
                   int64_t i0, int64_t i1, int64_t i2, int64_t i3) {
    switch (op) {
    case OP_FWD:        return fwd_elem(g, a, b, i0, i1, i2, i3);
    case OP_BWD_DATA:   return bwd_data_elem(g, a, b, i0, i1, i2, i3);
    case OP_BWD_WEIGHT: return bwd_weight_elem(g, a, b, i0, i1, i2, i3);
    default:            return convt_elem(g, a, b, i0, i1, i2, i3);
    }
}

static void unflatten(const int64_t d[4], int64_t f, int64_t idx[4]) {
    idx[3] = f % d[3]; f /= d[3];
    idx[2] = f % d[2]; f /= d[2];
    idx[1] = f % d[1]; f /= d[1];
    idx[0] = f;
}

/* Shape-vector argument order shared by all exported entry points:
 * g6[] = {n,h,w,c,k,r,s,sh,sw,ph,pw}. Operand a/b by op:
 *   fwd (x, W)   bwd_data (dy, W)   bwd_weight (x, dy)   convT (x, Wt)       */
static ocs make(const int64_t *v) {
    ocs g = {v[0], v[1], v[2], v[3], v[4], v[5], v[6], v[7], v[8], v[9], v[10]};
    return g;
}

void oracle_conv_out_dims(const int64_t *shape, int op, int64_t *dims) {
    ocs g = make(shape);
    out_dims(&g, op, dims);
}

void oracle_conv_full(const int64_t *shape, int op, const double *a,
                      const double *b, double *out) {
    ocs g = make(shape);
    int64_t d[4];
    out_dims(&g, op, d);
    int64_t total = d[0] * d[1] * d[2] * d[3];
#pragma omp parallel for schedule(dynamic, 256)
    for (int64_t f = 0; f < total; ++f) {
        int64_t i[4];
        unflatten(d, f, i);
        out[f] = elem(&g, op, a, b, i[0], i[1], i[2], i[3]);
    }
}

void oracle_conv_points(const int64_t *shape, int op, const double *a,
                        const double *b, int64_t npts, const int64_t *flat,
                        double *out) {
    ocs g = make(shape);
    int64_t d[4];
    out_dims(&g, op, d);
#pragma omp parallel for schedule(dynamic, 4)
    for (int64_t t = 0; t < npts; ++t) {
        int64_t i[4];
        unflatten(d, flat[t], i);
        out[t] = elem(&g, op, a, b, i[0], i[1], i[2], i[3]);
    }
}
