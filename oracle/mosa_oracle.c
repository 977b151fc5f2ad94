/*
 * Mixture of Sparse Attention (MoSA) layer -- plain CPU oracle in fp64.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg load this library.  The GPU path never calls
 * it, and the two share no source, header, table or helper.
 *
 * What is computed (paper, Section 2.2 "Mixture of Sparse Attention",
 * Eq. 1 attention, Eq. 2 multi-head sum, Eq. 3 MoSA layer), for every batch
 * element b and every MoSA head h independently (Section 2.1, expert-choice
 * footnote: the selection is made separately for each batch element):
 *
 *   s_t    = X_t . W^r                 router logit (Section 2.2), summed
 *                                      exactly and rounded once to double
 *   I      = the k tokens that come first under (s desc, t asc)
 *            (TopK of r = sigmoid(s): sigmoid is strictly increasing, so
 *            selecting on s is the same selection; ties -> lower index);
 *            reported in ascending order
 *   r_i    = sigmoid(s_{I_i}) = 1 / (1 + e^{-s})
 *   X^s    = X[I]                      (gather, Section 2.2)
 *   Q,K,V  = X^s W^Q, X^s W^K, X^s W^V
 *   A      = softmax((Q K^T + M) / sqrt(h')) V       (Eq. 1)
 *            M_ij = 0 iff I_i >= I_j (index-aware causal mask), else -inf;
 *            without the causal flag M = 0
 *   X^o    = diag(r) A W^O             (rows of A scaled by r^topk)
 *   Y_h[I_i] = X^o_i, other rows 0     (scatter, Section 2.2)
 *   Y      = sum_h Y_h  (Eq. 3, heads in ascending order)
 *            + sum over dense causal heads (Eq. 2; hybrid layer,
 *              "Hybridization" paragraph), i.e. heads with I = 0..T-1, r = 1.
 *
 * Variants of the layer (orc_options; all off by default):
 *   first_token  - every MoSA head always takes token 0 and chooses the other
 *                  k - 1 among t >= 1 by router score; token 0 is scaled by
 *                  its own r like any other (Section 3.2, IsoFLOP setting)
 *   fixed_stride - fixed sparse attention as a special case of MoSA:
 *                  I = 0, rho, 2 rho, ... and r = 1, no router (Section 3.1,
 *                  "Fixed Sparse Attention")
 *   rope         - rotary position encoding of q and k after the projections,
 *                  at the original positions I (Section 2.2, "Positional
 *                  encodings"); the first dh/2 dimensions are rotated in
 *                  adjacent pairs (2j, 2j+1) by angle p base^(-2j/(dh/2)), the
 *                  other half is left unchanged
 *   window       - the dense heads are local (sliding-window) causal heads:
 *                  query t sees keys t - window + 1 .. t (Section 3.4)
 *
 * Backward: the chain rule through the same expressions with I held fixed
 * (TopK is piecewise constant; the router receives its gradient through r,
 * Section 2.2 last paragraph), sigma'(s) = r (1 - r).
 *
 * Arithmetic: every input value (bf16 or fp32) is widened exactly to double.
 * All arithmetic is plain double.  Router logits are summed exactly
 * (Shewchuk's non-overlapping expansion sum with a final correctly rounded
 * result, Shewchuk 1997, "Adaptive Precision Floating-Point Arithmetic and
 * Fast Robust Geometric Predicates"): products of two bf16 or two fp32
 * numbers are exact in double, so the selection key is RN64(exact s).
 *
 * Determinism: per-(b,h) work may run on several OpenMP threads, but every
 * sum that crosses (b,h) tasks is done afterwards in a fixed order, so the
 * result does not depend on the thread count.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* Storage types of the inputs.  ORC_F64 exists only for the oracle's own
 * finite-difference checks; for it the router products are rounded, so the
 * "exact key" statement above holds for ORC_F32 and ORC_BF16 only. */
enum { ORC_F32 = 0, ORC_BF16 = 1, ORC_F64 = 2 };
enum { ORC_OK = 0, ORC_EINVAL = -1, ORC_ENOMEM = -2, ORC_EEXPANSION = -3 };

/* Layer variants (see the header comment); NULL means all off. */
typedef struct orc_options {
    int32_t first_token;
    int32_t fixed_stride;
    int32_t rope;
    int32_t window;
    double rope_base;
} orc_options;

static const orc_options orc_defaults = {0, 0, 0, 0, 10000.0};

/* ------------------------------------------------------------------------ */
/* Input widening                                                            */
/* ------------------------------------------------------------------------ */

static double widen_one(const void* p, int dtype, size_t i) {
    if (dtype == ORC_F32) return (double)((const float*)p)[i];
    if (dtype == ORC_F64) return ((const double*)p)[i];
    /* bf16: the upper 16 bits of an IEEE binary32 value. */
    uint32_t bits = (uint32_t)((const uint16_t*)p)[i] << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

static double* widen_all(const void* p, int dtype, size_t n) {
    double* out = (double*)malloc((n ? n : 1) * sizeof(double));
    if (!out) return NULL;
    for (size_t i = 0; i < n; ++i) out[i] = widen_one(p, dtype, i);
    return out;
}

/* ------------------------------------------------------------------------ */
/* Exact summation (Shewchuk expansion, correctly rounded result)            */
/* ------------------------------------------------------------------------ */

/* A sum held exactly as non-overlapping doubles of increasing magnitude.
 * A binary64 expansion never needs more than about 40 components. */
#define ORC_MAX_PARTS 96
typedef struct {
    double part[ORC_MAX_PARTS];
    int n;
    int overflow; /* set if the component bound was ever exceeded */
} exact_sum;

static void exact_sum_add(exact_sum* s, double x) {
    int kept = 0;
    for (int j = 0; j < s->n; ++j) {
        double y = s->part[j];
        if (fabs(x) < fabs(y)) { double t = x; x = y; y = t; }
        /* Fast two-sum (|x| >= |y|): hi + lo == x + y exactly. */
        double hi = x + y;
        double lo = y - (hi - x);
        if (lo != 0.0) s->part[kept++] = lo;
        x = hi;
    }
    if (kept >= ORC_MAX_PARTS) { s->overflow = 1; kept = ORC_MAX_PARTS - 1; }
    s->part[kept++] = x;
    s->n = kept;
}

/* Round the exact value of the expansion to the nearest double (ties to even). */
static double exact_sum_round(const exact_sum* s) {
    int n = s->n;
    if (n == 0) return 0.0;
    double hi = s->part[--n];
    double lo = 0.0;
    /* Add components from the largest down while the running sum stays exact. */
    while (n > 0) {
        double x = hi;
        double y = s->part[--n];
        hi = x + y;
        lo = y - (hi - x);
        if (lo != 0.0) break;
    }
    /* hi is RN(hi + lo).  If lo is exactly half an ulp (a tie), the components
     * still below it decide the direction: when they have the same sign as lo,
     * the true value lies past the midpoint and hi must step to hi + 2 lo. */
    if (n > 0 && ((lo < 0.0 && s->part[n - 1] < 0.0) || (lo > 0.0 && s->part[n - 1] > 0.0))) {
        double twice = lo * 2.0;
        double moved = hi + twice;
        if (moved - hi == twice) hi = moved;
    }
    return hi;
}

int orc_fsum(const double* v, int64_t n, double* out) {
    if (!v || !out || n < 0) return ORC_EINVAL;
    exact_sum s;
    s.n = 0;
    s.overflow = 0;
    for (int64_t i = 0; i < n; ++i) exact_sum_add(&s, v[i]);
    if (s.overflow) return ORC_EEXPANSION;
    *out = exact_sum_round(&s);
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Router keys and expert-choice TopK                                        */
/* ------------------------------------------------------------------------ */

/* keys[b,h,t] = RN64( sum_c X[b,t,c] * Wr[h,c] ), the sum taken exactly. */
int orc_router_keys(int dtype, int B, int T, int d, int H, const void* X, const void* Wr,
                    double* keys) {
    if (B < 1 || T < 1 || d < 1 || H < 1 || !X || !Wr || !keys) return ORC_EINVAL;
    int bad = 0;
#pragma omp parallel for schedule(dynamic) collapse(2) reduction(| : bad)
    for (int b = 0; b < B; ++b)
        for (int h = 0; h < H; ++h) {
            for (int t = 0; t < T; ++t) {
                exact_sum s;
                s.n = 0;
                s.overflow = 0;
                size_t xo = ((size_t)b * T + t) * d, wo = (size_t)h * d;
                for (int c = 0; c < d; ++c)
                    exact_sum_add(&s, widen_one(X, dtype, xo + c) * widen_one(Wr, dtype, wo + c));
                bad |= s.overflow;
                keys[((size_t)b * H + h) * T + t] = exact_sum_round(&s);
            }
        }
    return bad ? ORC_EEXPANSION : ORC_OK;
}

typedef struct {
    double key;
    int32_t t;
} candidate;

/* Total order of the expert-choice TopK: larger key first, then lower index. */
static int candidate_order(const void* pa, const void* pb) {
    const candidate* a = (const candidate*)pa;
    const candidate* b = (const candidate*)pb;
    if (a->key > b->key) return -1;
    if (a->key < b->key) return 1;
    return (a->t > b->t) - (a->t < b->t);
}

static int ascending_i32(const void* pa, const void* pb) {
    int32_t a = *(const int32_t*)pa, b = *(const int32_t*)pb;
    return (a > b) - (a < b);
}

/* The k tokens that come first under (key desc, t asc), written ascending.
 * first: token 0 is taken first and the other k - 1 come from t >= 1. */
static int select_row(int T, int k, int first, const double* key, int32_t* I) {
    candidate* c = (candidate*)malloc((size_t)T * sizeof(candidate));
    if (!c) return ORC_ENOMEM;
    const int t0 = first ? 1 : 0, n = T - t0;
    for (int t = t0; t < T; ++t) {
        c[t - t0].key = key[t];
        c[t - t0].t = t;
    }
    qsort(c, (size_t)n, sizeof(candidate), candidate_order);
    if (first) I[0] = 0;
    for (int i = t0; i < k; ++i) I[i] = c[i - t0].t;
    qsort(I, (size_t)k, sizeof(int32_t), ascending_i32);
    free(c);
    return ORC_OK;
}

int orc_select_ex(int B, int H, int T, int k, int first_token, const double* keys, int32_t* I) {
    if (B < 1 || H < 1 || T < 1 || k < 1 || k > T || !keys || !I) return ORC_EINVAL;
    int err = 0;
#pragma omp parallel for schedule(dynamic) reduction(| : err)
    for (int bh = 0; bh < B * H; ++bh)
        err |= select_row(T, k, first_token != 0, keys + (size_t)bh * T, I + (size_t)bh * k) ? 1 : 0;
    return err ? ORC_ENOMEM : ORC_OK;
}

int orc_select(int B, int H, int T, int k, const double* keys, int32_t* I) {
    return orc_select_ex(B, H, T, k, 0, keys, I);
}

/* Rotary encoding of one head vector v [dh] at position p (sign -1: the
 * inverse rotation, the transpose used by the backward pass).  The first
 * R = dh / 2 dimensions are rotated in pairs (2j, 2j+1), j < R / 2, by the
 * angle p theta_j with theta_j = base^(-2j/R); the rest stay as they are. */
static void rope_rotate(int dh, double base, double p, int sign, double* v) {
    const int R = dh / 2;
    for (int j = 0; j < R / 2; ++j) {
        const double theta = pow(base, -2.0 * j / R);
        const double a = sign * p * theta, c = cos(a), sn = sin(a);
        const double x = v[2 * j], y = v[2 * j + 1];
        v[2 * j] = x * c - y * sn;
        v[2 * j + 1] = x * sn + y * c;
    }
}

/* Exported for the oracle's own tests: rotate n vectors of dh at positions p. */
int orc_rope(int n, int dh, double base, const int32_t* p, int sign, double* v) {
    if (n < 0 || dh < 4 || dh % 4 || !(base > 1.0) || (sign != 1 && sign != -1) || !p || !v) return ORC_EINVAL;
    for (int i = 0; i < n; ++i) rope_rotate(dh, base, (double)p[i], sign, v + (size_t)i * dh);
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* One head on its selected tokens (Eq. 1 with the index-aware mask)         */
/* ------------------------------------------------------------------------ */

/* Intermediates of one head, kept for the backward pass. */
typedef struct {
    int n, d, dh;
    double *Xs, *Q, *K, *V, *P, *A; /* n*d, n*dh x3, n*n, n*dh */
} head_state;

static void head_state_free(head_state* s) {
    free(s->Xs); free(s->Q); free(s->K); free(s->V); free(s->P); free(s->A);
    memset(s, 0, sizeof *s);
}

static int head_state_alloc(head_state* s, int n, int d, int dh) {
    memset(s, 0, sizeof *s);
    s->n = n; s->d = d; s->dh = dh;
    s->Xs = (double*)malloc((size_t)n * d * sizeof(double));
    s->Q = (double*)malloc((size_t)n * dh * sizeof(double));
    s->K = (double*)malloc((size_t)n * dh * sizeof(double));
    s->V = (double*)malloc((size_t)n * dh * sizeof(double));
    s->P = (double*)malloc((size_t)n * n * sizeof(double));
    s->A = (double*)malloc((size_t)n * dh * sizeof(double));
    if (!s->Xs || !s->Q || !s->K || !s->V || !s->P || !s->A) {
        head_state_free(s);
        return ORC_ENOMEM;
    }
    return ORC_OK;
}

/* Q = Xs W for a [d, dh] weight. */
static void project(int n, int d, int dh, const double* Xs, const double* W, double* out) {
    for (int i = 0; i < n; ++i)
        for (int e = 0; e < dh; ++e) {
            double acc = 0.0;
            for (int c = 0; c < d; ++c) acc += Xs[(size_t)i * d + c] * W[(size_t)c * dh + e];
            out[(size_t)i * dh + e] = acc;
        }
}

/* Per-head attention options: the causal flag, the local window (dense
 * heads; 0 = none) and the rotary encoding (rope_base > 0) at positions I. */
typedef struct {
    int causal, window;
    double rope_base;
} head_opts;

static int may_attend(const head_opts* o, const int32_t* I, int i, int j) {
    if (o->causal && I[i] < I[j]) return 0;
    if (o->window > 0 && I[i] - I[j] >= o->window) return 0;
    return 1;
}

/* Forward of one head on the n tokens I (any order, no repeats).
 * Xb: [T, d] rows of one batch element; W*: [d, dh]; Wo: [dh, d].
 * Writes Xo[i, :] = r_i * A_i W^O for i < n.  r == NULL means r = 1. */
static void head_forward(int d, int dh, int n, const head_opts* o, const double* Xb, const double* Wq,
                         const double* Wk, const double* Wv, const double* Wo, const int32_t* I,
                         const double* r, head_state* s, double* Xo) {
    /* gather */
    for (int i = 0; i < n; ++i)
        memcpy(s->Xs + (size_t)i * d, Xb + (size_t)I[i] * d, (size_t)d * sizeof(double));
    /* projections */
    project(n, d, dh, s->Xs, Wq, s->Q);
    project(n, d, dh, s->Xs, Wk, s->K);
    project(n, d, dh, s->Xs, Wv, s->V);
    /* rotary encoding of q and k at the original positions I */
    if (o->rope_base > 0.0)
        for (int i = 0; i < n; ++i) {
            rope_rotate(dh, o->rope_base, (double)I[i], 1, s->Q + (size_t)i * dh);
            rope_rotate(dh, o->rope_base, (double)I[i], 1, s->K + (size_t)i * dh);
        }
    /* attention, Eq. 1: P = softmax((Q K^T + M) / sqrt(h')), computed max-subtracted */
    const double scale = 1.0 / sqrt((double)dh);
    for (int i = 0; i < n; ++i) {
        double* Pi = s->P + (size_t)i * n;
        double mx = -INFINITY;
        for (int j = 0; j < n; ++j) {
            if (!may_attend(o, I, i, j)) continue;
            double dot = 0.0;
            for (int e = 0; e < dh; ++e) dot += s->Q[(size_t)i * dh + e] * s->K[(size_t)j * dh + e];
            Pi[j] = dot * scale;
            if (Pi[j] > mx) mx = Pi[j];
        }
        double den = 0.0;
        for (int j = 0; j < n; ++j) {
            if (!may_attend(o, I, i, j)) { Pi[j] = 0.0; continue; }
            Pi[j] = exp(Pi[j] - mx);
            den += Pi[j];
        }
        for (int j = 0; j < n; ++j) Pi[j] /= den;
        for (int e = 0; e < dh; ++e) {
            double acc = 0.0;
            for (int j = 0; j < n; ++j) acc += Pi[j] * s->V[(size_t)j * dh + e];
            s->A[(size_t)i * dh + e] = acc;
        }
    }
    /* X^o = diag(r) A W^O */
    for (int i = 0; i < n; ++i) {
        double ri = r ? r[i] : 1.0;
        for (int c = 0; c < d; ++c) {
            double acc = 0.0;
            for (int e = 0; e < dh; ++e) acc += s->A[(size_t)i * dh + e] * Wo[(size_t)e * d + c];
            Xo[(size_t)i * d + c] = ri * acc;
        }
    }
}

/* Backward of one head given dXo = dY[I] (n x d).  Accumulates into the
 * per-head weight gradients (caller owns them, no sharing between threads),
 * writes dXs (n x d) and, when r != NULL, the router gradient into dWr. */
static void head_backward(int d, int dh, int n, const head_opts* o, const int32_t* I, const double* Wq,
                          const double* Wk, const double* Wv, const double* Wo, const double* Wr,
                          const double* r, const head_state* s, const double* dXo, double* dWq,
                          double* dWk, double* dWv, double* dWo, double* dWr, double* dXs) {
    const double scale = 1.0 / sqrt((double)dh);
    double* dAt = (double*)calloc((size_t)n * dh, sizeof(double)); /* d(diag(r) A) */
    double* dA = (double*)calloc((size_t)n * dh, sizeof(double));
    double* dP = (double*)calloc((size_t)n * n, sizeof(double));
    double* dQ = (double*)calloc((size_t)n * dh, sizeof(double));
    double* dK = (double*)calloc((size_t)n * dh, sizeof(double));
    double* dV = (double*)calloc((size_t)n * dh, sizeof(double));
    double* dz = (double*)calloc((size_t)n, sizeof(double));

    for (int i = 0; i < n; ++i) {
        double ri = r ? r[i] : 1.0;
        /* dW^O += (r_i A_i)^T dXo_i ; d(rA)_i = dXo_i W^O^T */
        for (int e = 0; e < dh; ++e) {
            double a = ri * s->A[(size_t)i * dh + e];
            double acc = 0.0;
            for (int c = 0; c < d; ++c) {
                dWo[(size_t)e * d + c] += a * dXo[(size_t)i * d + c];
                acc += dXo[(size_t)i * d + c] * Wo[(size_t)e * d + c];
            }
            dAt[(size_t)i * dh + e] = acc;
        }
        /* r_i scales row i: dr_i = <d(rA)_i, A_i>, dA_i = r_i d(rA)_i */
        double dr = 0.0;
        for (int e = 0; e < dh; ++e) {
            dr += dAt[(size_t)i * dh + e] * s->A[(size_t)i * dh + e];
            dA[(size_t)i * dh + e] = ri * dAt[(size_t)i * dh + e];
        }
        dz[i] = r ? dr * ri * (1.0 - ri) : 0.0;
    }
    /* A = P V */
    for (int j = 0; j < n; ++j)
        for (int e = 0; e < dh; ++e) {
            double acc = 0.0;
            for (int i = 0; i < n; ++i) acc += s->P[(size_t)i * n + j] * dA[(size_t)i * dh + e];
            dV[(size_t)j * dh + e] = acc;
        }
    for (int i = 0; i < n; ++i)
        for (int j = 0; j < n; ++j) {
            double acc = 0.0;
            for (int e = 0; e < dh; ++e) acc += dA[(size_t)i * dh + e] * s->V[(size_t)j * dh + e];
            dP[(size_t)i * n + j] = acc;
        }
    /* softmax rows: dS_ij = P_ij (dP_ij - sum_l P_il dP_il); masked entries have P = 0 */
    for (int i = 0; i < n; ++i) {
        double rowdot = 0.0;
        for (int j = 0; j < n; ++j) rowdot += s->P[(size_t)i * n + j] * dP[(size_t)i * n + j];
        for (int j = 0; j < n; ++j)
            dP[(size_t)i * n + j] = s->P[(size_t)i * n + j] * (dP[(size_t)i * n + j] - rowdot);
    }
    /* scores = Q K^T / sqrt(h') */
    for (int i = 0; i < n; ++i)
        for (int e = 0; e < dh; ++e) {
            double acc = 0.0;
            for (int j = 0; j < n; ++j) acc += dP[(size_t)i * n + j] * s->K[(size_t)j * dh + e];
            dQ[(size_t)i * dh + e] = acc * scale;
        }
    for (int j = 0; j < n; ++j)
        for (int e = 0; e < dh; ++e) {
            double acc = 0.0;
            for (int i = 0; i < n; ++i) acc += dP[(size_t)i * n + j] * s->Q[(size_t)i * dh + e];
            dK[(size_t)j * dh + e] = acc * scale;
        }
    /* through the rotation: d(X^s W^Q) = R(p)^T dQ, likewise for K */
    if (o->rope_base > 0.0)
        for (int i = 0; i < n; ++i) {
            rope_rotate(dh, o->rope_base, (double)I[i], -1, dQ + (size_t)i * dh);
            rope_rotate(dh, o->rope_base, (double)I[i], -1, dK + (size_t)i * dh);
        }
    /* projections Q = Xs W^Q etc., router s = Xs W^r */
    for (int c = 0; c < d; ++c) {
        for (int e = 0; e < dh; ++e) {
            double gq = 0.0, gk = 0.0, gv = 0.0;
            for (int i = 0; i < n; ++i) {
                double x = s->Xs[(size_t)i * d + c];
                gq += x * dQ[(size_t)i * dh + e];
                gk += x * dK[(size_t)i * dh + e];
                gv += x * dV[(size_t)i * dh + e];
            }
            dWq[(size_t)c * dh + e] += gq;
            dWk[(size_t)c * dh + e] += gk;
            dWv[(size_t)c * dh + e] += gv;
        }
        if (r) {
            double gr = 0.0;
            for (int i = 0; i < n; ++i) gr += dz[i] * s->Xs[(size_t)i * d + c];
            dWr[c] += gr;
        }
    }
    for (int i = 0; i < n; ++i)
        for (int c = 0; c < d; ++c) {
            double acc = r ? dz[i] * Wr[c] : 0.0;
            for (int e = 0; e < dh; ++e)
                acc += dQ[(size_t)i * dh + e] * Wq[(size_t)c * dh + e] +
                       dK[(size_t)i * dh + e] * Wk[(size_t)c * dh + e] +
                       dV[(size_t)i * dh + e] * Wv[(size_t)c * dh + e];
            dXs[(size_t)i * d + c] = acc;
        }
    free(dAt); free(dA); free(dP); free(dQ); free(dK); free(dV); free(dz);
}

/* Exported single-head entry: attention of one head over a given token set I
 * with given router values r (NULL = all ones).  All arrays are double.
 * Y [T, d] is ACCUMULATED: Y[I_i] += r_i A_i W^O. */
int orc_head_attend(int T, int d, int dh, int n, int causal, const double* Xb, const double* Wq,
                    const double* Wk, const double* Wv, const double* Wo, const int32_t* I,
                    const double* r, double* Y) {
    if (T < 1 || d < 1 || dh < 1 || n < 1 || n > T || !Xb || !Wq || !Wk || !Wv || !Wo || !I || !Y)
        return ORC_EINVAL;
    for (int i = 0; i < n; ++i)
        if (I[i] < 0 || I[i] >= T) return ORC_EINVAL;
    head_state s;
    if (head_state_alloc(&s, n, d, dh)) return ORC_ENOMEM;
    double* Xo = (double*)malloc((size_t)n * d * sizeof(double));
    if (!Xo) { head_state_free(&s); return ORC_ENOMEM; }
    const head_opts o = {causal, 0, 0.0};
    head_forward(d, dh, n, &o, Xb, Wq, Wk, Wv, Wo, I, r, &s, Xo);
    for (int i = 0; i < n; ++i)
        for (int c = 0; c < d; ++c) Y[(size_t)I[i] * d + c] += Xo[(size_t)i * d + c];
    free(Xo);
    head_state_free(&s);
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Whole layer                                                               */
/* ------------------------------------------------------------------------ */

typedef struct {
    int dtype, B, T, d, H, dh, k, causal, Hd;
    orc_options opt;
} layer_shape;

/* Attention options of the MoSA heads and of the dense heads. */
static head_opts mosa_opts(const layer_shape* L) {
    head_opts o = {L->causal, 0, L->opt.rope ? L->opt.rope_base : 0.0};
    return o;
}
static head_opts dense_opts(const layer_shape* L) {
    head_opts o = {L->causal, L->opt.window, L->opt.rope ? L->opt.rope_base : 0.0};
    return o;
}

typedef struct {
    double *Wr, *Wq, *Wk, *Wv, *Wo;     /* MoSA heads */
    double *Wqd, *Wkd, *Wvd, *Wod;      /* dense heads (may be NULL when Hd == 0) */
} layer_weights;

static void weights_free(layer_weights* w) {
    free(w->Wr); free(w->Wq); free(w->Wk); free(w->Wv); free(w->Wo);
    free(w->Wqd); free(w->Wkd); free(w->Wvd); free(w->Wod);
    memset(w, 0, sizeof *w);
}

static int weights_widen(const layer_shape* L, const void* Wr, const void* Wq, const void* Wk,
                         const void* Wv, const void* Wo, const void* Wqd, const void* Wkd,
                         const void* Wvd, const void* Wod, layer_weights* w) {
    memset(w, 0, sizeof *w);
    size_t proj = (size_t)L->d * L->dh;
    if (L->H > 0) {
        /* fixed sparse attention has no router: W^r may be NULL */
        w->Wr = Wr ? widen_all(Wr, L->dtype, (size_t)L->H * L->d) : (double*)calloc((size_t)L->H * L->d, sizeof(double));
        w->Wq = widen_all(Wq, L->dtype, (size_t)L->H * proj);
        w->Wk = widen_all(Wk, L->dtype, (size_t)L->H * proj);
        w->Wv = widen_all(Wv, L->dtype, (size_t)L->H * proj);
        w->Wo = widen_all(Wo, L->dtype, (size_t)L->H * proj);
        if (!w->Wr || !w->Wq || !w->Wk || !w->Wv || !w->Wo) goto fail;
    }
    if (L->Hd > 0) {
        w->Wqd = widen_all(Wqd, L->dtype, (size_t)L->Hd * proj);
        w->Wkd = widen_all(Wkd, L->dtype, (size_t)L->Hd * proj);
        w->Wvd = widen_all(Wvd, L->dtype, (size_t)L->Hd * proj);
        w->Wod = widen_all(Wod, L->dtype, (size_t)L->Hd * proj);
        if (!w->Wqd || !w->Wkd || !w->Wvd || !w->Wod) goto fail;
    }
    return ORC_OK;
fail:
    weights_free(w);
    return ORC_ENOMEM;
}

static int shape_ok(const layer_shape* L, const void* X, const void* Wr, const void* Wq,
                    const void* Wk, const void* Wv, const void* Wo, const void* Wqd,
                    const void* Wkd, const void* Wvd, const void* Wod) {
    if (L->dtype != ORC_F32 && L->dtype != ORC_BF16 && L->dtype != ORC_F64) return 0;
    if (L->B < 1 || L->T < 1 || L->d < 1 || L->dh < 1 || L->H < 0 || L->Hd < 0) return 0;
    if (L->H + L->Hd < 1 || !X) return 0;
    if (L->H > 0 && (L->k < 1 || L->k > L->T || !Wq || !Wk || !Wv || !Wo)) return 0;
    if (L->H > 0 && !Wr && L->opt.fixed_stride <= 0) return 0;
    if (L->Hd > 0 && (!Wqd || !Wkd || !Wvd || !Wod)) return 0;
    const orc_options* o = &L->opt;
    if (o->fixed_stride < 0 || o->window < 0 || (o->rope && !(o->rope_base > 1.0))) return 0;
    if (o->rope && L->dh % 4) return 0;
    if (o->fixed_stride > 0 && (o->first_token || (double)(L->k - 1) * o->fixed_stride > L->T - 1)) return 0;
    return 1;
}

/* Selection for every (b,h): I [B,H,k] ascending, r [B,H,k], keys [B,H,T]. */
static int layer_select(const layer_shape* L, const void* X, const void* Wr, double* keys,
                        int32_t* I, double* r) {
    if (L->opt.fixed_stride > 0) {
        /* I = 0, rho, 2 rho, ...; r = 1; no router (keys reported as 0) */
        memset(keys, 0, (size_t)L->B * L->H * L->T * sizeof(double));
        for (size_t bh = 0; bh < (size_t)L->B * L->H; ++bh)
            for (int i = 0; i < L->k; ++i) {
                I[bh * L->k + i] = i * L->opt.fixed_stride;
                r[bh * L->k + i] = 1.0;
            }
        return ORC_OK;
    }
    int e = orc_router_keys(L->dtype, L->B, L->T, L->d, L->H, X, Wr, keys);
    if (e) return e;
    e = orc_select_ex(L->B, L->H, L->T, L->k, L->opt.first_token, keys, I);
    if (e) return e;
    for (size_t bh = 0; bh < (size_t)L->B * L->H; ++bh)
        for (int i = 0; i < L->k; ++i) {
            double s = keys[bh * L->T + I[bh * L->k + i]];
            r[bh * L->k + i] = 1.0 / (1.0 + exp(-s));
        }
    return ORC_OK;
}

/* Forward of the layer.  Y [B,T,d] (written, not accumulated).
 * Optional outputs (NULL to skip): I_out [B,H,k], r_out [B,H,k],
 * keys_out [B,H,T], and the per-head intermediates of the MoSA heads
 * Q_out, K_out, V_out, A_out [B,H,k,dh] (A before the router scaling). */
int orc_forward_ex(int dtype, int B, int T, int d, int H, int dh, int k, int causal, int Hd,
                   const void* X, const void* Wr, const void* Wq, const void* Wk, const void* Wv,
                   const void* Wo, const void* Wqd, const void* Wkd, const void* Wvd,
                   const void* Wod, double* Y, int32_t* I_out, double* r_out, double* keys_out,
                   double* Q_out, double* K_out, double* V_out, double* A_out, const orc_options* opt) {
    layer_shape L = {dtype, B, T, d, H, dh, k, causal, Hd, opt ? *opt : orc_defaults};
    if (!shape_ok(&L, X, Wr, Wq, Wk, Wv, Wo, Wqd, Wkd, Wvd, Wod) || !Y) return ORC_EINVAL;
    const size_t proj = (size_t)d * dh;
    int err = ORC_ENOMEM;
    layer_weights w;
    double* Xd = widen_all(X, dtype, (size_t)B * T * d);
    if (!Xd) return ORC_ENOMEM;
    if (weights_widen(&L, Wr, Wq, Wk, Wv, Wo, Wqd, Wkd, Wvd, Wod, &w)) { free(Xd); return ORC_ENOMEM; }

    const size_t nsel = (size_t)B * H * (H > 0 ? k : 0);
    double* keys = (double*)malloc(((size_t)B * H * T + 1) * sizeof(double));
    int32_t* I = (int32_t*)malloc((nsel + 1) * sizeof(int32_t));
    double* r = (double*)malloc((nsel + 1) * sizeof(double));
    /* contributions X^o of every MoSA head (B*H*k rows) and dense head (B*Hd*T rows) */
    double* XoM = (double*)malloc((nsel * d + 1) * sizeof(double));
    double* XoD = (double*)malloc(((size_t)B * Hd * T * d + 1) * sizeof(double));
    int32_t* iota = (int32_t*)malloc((size_t)T * sizeof(int32_t));
    if (!keys || !I || !r || !XoM || !XoD || !iota) goto done;
    for (int t = 0; t < T; ++t) iota[t] = t;

    if (H > 0) {
        err = layer_select(&L, X, Wr, keys, I, r);
        if (err) goto done;
    }
    int fail = 0;
    /* MoSA heads: independent (b,h) tasks */
#pragma omp parallel for schedule(dynamic) reduction(| : fail)
    for (int bh = 0; bh < B * H; ++bh) {
        int b = bh / H, h = bh % H;
        head_state s;
        if (head_state_alloc(&s, k, d, dh)) { fail |= 1; continue; }
        const head_opts o = mosa_opts(&L);
        head_forward(d, dh, k, &o, Xd + (size_t)b * T * d, w.Wq + h * proj, w.Wk + h * proj,
                     w.Wv + h * proj, w.Wo + h * proj, I + (size_t)bh * k, r + (size_t)bh * k, &s,
                     XoM + (size_t)bh * k * d);
        size_t qo = (size_t)bh * k * dh;
        if (Q_out) memcpy(Q_out + qo, s.Q, (size_t)k * dh * sizeof(double));
        if (K_out) memcpy(K_out + qo, s.K, (size_t)k * dh * sizeof(double));
        if (V_out) memcpy(V_out + qo, s.V, (size_t)k * dh * sizeof(double));
        if (A_out) memcpy(A_out + qo, s.A, (size_t)k * dh * sizeof(double));
        head_state_free(&s);
    }
    /* dense heads: I = 0..T-1, r = 1 */
#pragma omp parallel for schedule(dynamic) reduction(| : fail)
    for (int bh = 0; bh < B * Hd; ++bh) {
        int b = bh / Hd, h = bh % Hd;
        head_state s;
        if (head_state_alloc(&s, T, d, dh)) { fail |= 1; continue; }
        const head_opts o = dense_opts(&L);
        head_forward(d, dh, T, &o, Xd + (size_t)b * T * d, w.Wqd + h * proj, w.Wkd + h * proj,
                     w.Wvd + h * proj, w.Wod + h * proj, iota, NULL, &s,
                     XoD + (size_t)bh * T * d);
        head_state_free(&s);
    }
    if (fail) { err = ORC_ENOMEM; goto done; }
    /* Eq. 3 sum: per batch element, MoSA heads in ascending order, then dense heads */
#pragma omp parallel for schedule(static)
    for (int b = 0; b < B; ++b) {
        double* Yb = Y + (size_t)b * T * d;
        memset(Yb, 0, (size_t)T * d * sizeof(double));
        for (int h = 0; h < H; ++h) {
            size_t bh = (size_t)b * H + h;
            for (int i = 0; i < k; ++i) {
                const double* src = XoM + (bh * k + i) * d;
                double* dst = Yb + (size_t)I[bh * k + i] * d;
                for (int c = 0; c < d; ++c) dst[c] += src[c];
            }
        }
        for (int h = 0; h < Hd; ++h) {
            const double* src = XoD + ((size_t)b * Hd + h) * T * d;
            for (size_t e = 0; e < (size_t)T * d; ++e) Yb[e] += src[e];
        }
    }
    if (I_out) memcpy(I_out, I, nsel * sizeof(int32_t));
    if (r_out) memcpy(r_out, r, nsel * sizeof(double));
    if (keys_out) memcpy(keys_out, keys, (size_t)B * H * T * sizeof(double));
    err = ORC_OK;
done:
    free(keys); free(I); free(r); free(XoM); free(XoD); free(iota); free(Xd);
    weights_free(&w);
    return err;
}

/* Backward of the layer for upstream gradient dY [B,T,d] (dtype of X).
 * Outputs (double, written not accumulated): dX [B,T,d], dWr [H,d],
 * dWq/dWk/dWv [H,d,dh], dWo [H,dh,d], and the dense-head gradients
 * dWqd/dWkd/dWvd [Hd,d,dh], dWod [Hd,dh,d] (NULL allowed when Hd == 0). */
int orc_backward_ex(int dtype, int B, int T, int d, int H, int dh, int k, int causal, int Hd,
                    const void* X, const void* Wr, const void* Wq, const void* Wk, const void* Wv,
                    const void* Wo, const void* Wqd, const void* Wkd, const void* Wvd,
                    const void* Wod, const void* dY, double* dX, double* dWr, double* dWq,
                    double* dWk, double* dWv, double* dWo, double* dWqd, double* dWkd, double* dWvd,
                    double* dWod, const orc_options* opt) {
    layer_shape L = {dtype, B, T, d, H, dh, k, causal, Hd, opt ? *opt : orc_defaults};
    if (!shape_ok(&L, X, Wr, Wq, Wk, Wv, Wo, Wqd, Wkd, Wvd, Wod) || !dY || !dX) return ORC_EINVAL;
    if (H > 0 && (!dWr || !dWq || !dWk || !dWv || !dWo)) return ORC_EINVAL;
    if (Hd > 0 && (!dWqd || !dWkd || !dWvd || !dWod)) return ORC_EINVAL;
    const size_t proj = (size_t)d * dh;
    int err = ORC_ENOMEM;
    layer_weights w;
    double* Xd = widen_all(X, dtype, (size_t)B * T * d);
    double* dYd = widen_all(dY, dtype, (size_t)B * T * d);
    if (!Xd || !dYd) { free(Xd); free(dYd); return ORC_ENOMEM; }
    if (weights_widen(&L, Wr, Wq, Wk, Wv, Wo, Wqd, Wkd, Wvd, Wod, &w)) {
        free(Xd); free(dYd);
        return ORC_ENOMEM;
    }
    const size_t nsel = (size_t)B * H * (H > 0 ? k : 0);
    double* keys = (double*)malloc(((size_t)B * H * T + 1) * sizeof(double));
    int32_t* I = (int32_t*)malloc((nsel + 1) * sizeof(int32_t));
    double* r = (double*)malloc((nsel + 1) * sizeof(double));
    double* dXsM = (double*)malloc((nsel * d + 1) * sizeof(double));
    double* dXsD = (double*)malloc(((size_t)B * Hd * T * d + 1) * sizeof(double));
    int32_t* iota = (int32_t*)malloc((size_t)T * sizeof(int32_t));
    if (!keys || !I || !r || !dXsM || !dXsD || !iota) goto done;
    for (int t = 0; t < T; ++t) iota[t] = t;
    if (H > 0) {
        err = layer_select(&L, X, Wr, keys, I, r);
        if (err) goto done;
        memset(dWr, 0, (size_t)H * d * sizeof(double));
        memset(dWq, 0, (size_t)H * proj * sizeof(double));
        memset(dWk, 0, (size_t)H * proj * sizeof(double));
        memset(dWv, 0, (size_t)H * proj * sizeof(double));
        memset(dWo, 0, (size_t)H * proj * sizeof(double));
    }
    if (Hd > 0) {
        memset(dWqd, 0, (size_t)Hd * proj * sizeof(double));
        memset(dWkd, 0, (size_t)Hd * proj * sizeof(double));
        memset(dWvd, 0, (size_t)Hd * proj * sizeof(double));
        memset(dWod, 0, (size_t)Hd * proj * sizeof(double));
    }
    int fail = 0;
    /* One task per head; inside it the batch elements are visited in order,
     * so the weight-gradient sums over b have a fixed order. */
#pragma omp parallel for schedule(dynamic) reduction(| : fail)
    for (int h = 0; h < H; ++h) {
        head_state s;
        double* dXo = (double*)malloc((size_t)k * d * sizeof(double));
        double* Xo = (double*)malloc((size_t)k * d * sizeof(double));
        if (!dXo || !Xo || head_state_alloc(&s, k, d, dh)) { fail |= 1; free(dXo); free(Xo); continue; }
        const head_opts o = mosa_opts(&L);
        /* fixed sparse attention: r = 1 and no router gradient */
        const int routed = L.opt.fixed_stride <= 0;
        for (int b = 0; b < B; ++b) {
            size_t bh = (size_t)b * H + h;
            const int32_t* Ib = I + bh * k;
            head_forward(d, dh, k, &o, Xd + (size_t)b * T * d, w.Wq + h * proj,
                         w.Wk + h * proj, w.Wv + h * proj, w.Wo + h * proj, Ib, r + bh * k, &s, Xo);
            for (int i = 0; i < k; ++i)
                memcpy(dXo + (size_t)i * d, dYd + ((size_t)b * T + Ib[i]) * d, (size_t)d * sizeof(double));
            head_backward(d, dh, k, &o, Ib, w.Wq + h * proj, w.Wk + h * proj, w.Wv + h * proj,
                          w.Wo + h * proj, w.Wr + (size_t)h * d, routed ? r + bh * k : NULL, &s, dXo,
                          dWq + h * proj, dWk + h * proj, dWv + h * proj, dWo + h * proj,
                          dWr + (size_t)h * d, dXsM + bh * k * d);
        }
        head_state_free(&s);
        free(dXo); free(Xo);
    }
#pragma omp parallel for schedule(dynamic) reduction(| : fail)
    for (int h = 0; h < Hd; ++h) {
        head_state s;
        double* dXo = (double*)malloc((size_t)T * d * sizeof(double));
        double* Xo = (double*)malloc((size_t)T * d * sizeof(double));
        if (!dXo || !Xo || head_state_alloc(&s, T, d, dh)) { fail |= 1; free(dXo); free(Xo); continue; }
        const head_opts o = dense_opts(&L);
        for (int b = 0; b < B; ++b) {
            size_t bh = (size_t)b * Hd + h;
            head_forward(d, dh, T, &o, Xd + (size_t)b * T * d, w.Wqd + h * proj,
                         w.Wkd + h * proj, w.Wvd + h * proj, w.Wod + h * proj, iota, NULL, &s, Xo);
            memcpy(dXo, dYd + (size_t)b * T * d, (size_t)T * d * sizeof(double));
            head_backward(d, dh, T, &o, iota, w.Wqd + h * proj, w.Wkd + h * proj, w.Wvd + h * proj,
                          w.Wod + h * proj, NULL, NULL, &s, dXo, dWqd + h * proj, dWkd + h * proj,
                          dWvd + h * proj, dWod + h * proj, NULL, dXsD + bh * T * d);
        }
        head_state_free(&s);
        free(dXo); free(Xo);
    }
    if (fail) { err = ORC_ENOMEM; goto done; }
    /* dX: scatter-add per batch element, MoSA heads ascending, then dense heads */
#pragma omp parallel for schedule(static)
    for (int b = 0; b < B; ++b) {
        double* dXb = dX + (size_t)b * T * d;
        memset(dXb, 0, (size_t)T * d * sizeof(double));
        for (int h = 0; h < H; ++h) {
            size_t bh = (size_t)b * H + h;
            for (int i = 0; i < k; ++i) {
                const double* src = dXsM + (bh * k + i) * d;
                double* dst = dXb + (size_t)I[bh * k + i] * d;
                for (int c = 0; c < d; ++c) dst[c] += src[c];
            }
        }
        for (int h = 0; h < Hd; ++h) {
            const double* src = dXsD + ((size_t)b * Hd + h) * T * d;
            for (size_t e = 0; e < (size_t)T * d; ++e) dXb[e] += src[e];
        }
    }
    err = ORC_OK;
done:
    free(keys); free(I); free(r); free(dXsM); free(dXsD); free(iota); free(Xd); free(dYd);
    weights_free(&w);
    return err;
}

int orc_forward(int dtype, int B, int T, int d, int H, int dh, int k, int causal, int Hd,
                const void* X, const void* Wr, const void* Wq, const void* Wk, const void* Wv,
                const void* Wo, const void* Wqd, const void* Wkd, const void* Wvd,
                const void* Wod, double* Y, int32_t* I_out, double* r_out, double* keys_out,
                double* Q_out, double* K_out, double* V_out, double* A_out) {
    return orc_forward_ex(dtype, B, T, d, H, dh, k, causal, Hd, X, Wr, Wq, Wk, Wv, Wo, Wqd, Wkd, Wvd, Wod, Y,
                          I_out, r_out, keys_out, Q_out, K_out, V_out, A_out, NULL);
}

int orc_backward(int dtype, int B, int T, int d, int H, int dh, int k, int causal, int Hd,
                 const void* X, const void* Wr, const void* Wq, const void* Wk, const void* Wv,
                 const void* Wo, const void* Wqd, const void* Wkd, const void* Wvd,
                 const void* Wod, const void* dY, double* dX, double* dWr, double* dWq,
                 double* dWk, double* dWv, double* dWo, double* dWqd, double* dWkd, double* dWvd,
                 double* dWod) {
    return orc_backward_ex(dtype, B, T, d, H, dh, k, causal, Hd, X, Wr, Wq, Wk, Wv, Wo, Wqd, Wkd, Wvd, Wod, dY,
                           dX, dWr, dWq, dWk, dWv, dWo, dWqd, dWkd, dWvd, dWod, NULL);
}

int orc_max_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

void orc_set_threads(int n) {
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}
