/*
 * KVarN CPU oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, obviously-correct fp64 implementation of what the KVarN hot path
 * computes (KVarN: Variance-Normalized KV-Cache Quantization, arXiv 2606.03458):
 *   - per-token Hadamard rotation along head_dim            (Sec. 2.2, Sec. 3.3, App. A)
 *   - VarN, alternating log-domain dual-scale balancing     (Sec. 3.3, App. H, Algorithm 1)
 *   - KIVI-style asymmetric round-to-nearest per group      (Sec. 2.1, Eq. 1)
 *   - dual-scale storage with the Sinkhorn scale absorbed   (App. D "Effective memory overhead")
 *   - decode attention over sink + quantized body + residual (App. D "Quantization", App. I)
 *
 * Only the test-suite, the smoke check and the benchmark's CPU-baseline leg may load this
 * library.  It shares no code, header, table or helper with the GPU library: the packed
 * tile format is implemented here a second time, from its written description.
 *
 * Every floating-point step runs in double precision.  Values that the format stores in
 * fp32 (the three auxiliary vectors) are rounded once, to nearest-even, when stored.  The
 * compact format of App. D ("Effective memory overhead": per group of 128 values, the two
 * scales in an 8-bit float format and the zero point in a 16-bit one) rounds them to OCP E4M3
 * and IEEE binary16 instead, see kvo_quantize_tile.
 *
 * Parity pins for each function live in tests/test_oracle_*.py.  The constants c_min and
 * c_max of Algorithm 1 are not given numerically by the paper (parity unpinned; 1e-8 and
 * 1e8 by default, see the params struct).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define D 128   /* head_dim: channels per token                       (Sec. 2.1) */
#define G 128   /* tokens per quantization group / block              (Sec. 2.1, App. D) */

enum { KVO_KEYS = 0, KVO_VALUES = 1 };

typedef struct {
    int32_t bits;        /* 2 or 4 */
    int32_t varn_iters;  /* K of Algorithm 1 (8 in the runtime experiment, Sec. 4.2) */
    double c_min, c_max; /* variance clamp of Algorithm 1 (values unstated in the paper) */
    double log_lo, log_hi; /* clamp of the cumulative log-scales: -0.3 and 10.0 in Algorithm 1 */
    double imb_floor;    /* floor on min variance inside Imb(): 1e-8 in Algorithm 1 */
    int32_t ddof;        /* variance estimator: 1 (unbiased) by default */
    int32_t aux;         /* stored aux format: 0 = three fp32 vectors, 1 = compact (E4M3 a and s2,
                            binary16 b) */
    int32_t force_best;  /* -1: Algorithm 1's selection.  k in 0..K: keep iteration k's scales
                            instead (test use: the outcome had iteration k won a near-tie) */
    int32_t rotate;      /* 1: Hadamard rotation before VarN (KVarN); 0: none (the ablations of
                            Fig. 1: KIVI-style RTN with K = 0, VarN alone with K > 0) */
} kvo_params;

/* ------------------------------------------------------------------------------------------
 * bf16 <-> double.  bf16 is the upper half of an IEEE binary32.
 * ------------------------------------------------------------------------------------------ */
double kvo_bf16_to_double(uint16_t h) {
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, 4);
    return (double)f;
}

/* Round a double to bf16, nearest-even (via binary32, then binary32 -> bf16 nearest-even).
 * Used only to store outputs; NaN is not produced by the oracle's inputs. */
uint16_t kvo_double_to_bf16(double x) {
    float f = (float)x;
    uint32_t u;
    memcpy(&u, &f, 4);
    uint32_t lsb = (u >> 16) & 1u;
    u += 0x7FFFu + lsb;
    return (uint16_t)(u >> 16);
}

/* ------------------------------------------------------------------------------------------
 * Narrow formats of the compact aux (App. D, "Effective memory overhead": 8-bit float scales,
 * a 16-bit float zero point).
 *   E4M3 (the OCP 8-bit floating-point format E4M3): sign, 4 exponent bits with bias 7, 3
 *   mantissa bits.  Exponent field 0 holds the subnormals m * 2^-9; there are no infinities and
 *   the pattern with all exponent and mantissa bits set is NaN, so the largest finite value is
 *   1.75 * 2^8 = 448.  Only positive values are stored here (scales).
 *   binary16 (IEEE 754): 5 exponent bits with bias 15, 10 mantissa bits, subnormals
 *   m * 2^-24, largest finite 65504.
 * Encoding rounds on the grid of the binade of x (spacing 2^(e - mantissa bits), subnormal
 * spacing below the smallest normal): to nearest with ties to the even grid point, or upward.
 * Values beyond the largest finite one saturate to it.
 * ------------------------------------------------------------------------------------------ */
double kvo_e4m3_to_double(uint8_t v) {
    const int e = (v >> 3) & 15, m = v & 7;
    const double mag = e == 0 ? ldexp((double)m, -9) : ldexp(1.0 + m / 8.0, e - 7);
    return (v & 0x80) ? -mag : mag;
}

uint8_t kvo_e4m3_from_double(double x, int round_up) {
    if (!(x > 0.0)) return 0;
    if (x >= 448.0) return 0x7E; /* exponent field 15, mantissa 6: 448 */
    int ex;
    frexp(x, &ex); /* x = f * 2^ex, f in [0.5, 1): binade [2^(ex-1), 2^ex) */
    int E = ex - 1;
    if (E < -6) E = -6; /* subnormal grid spacing 2^-9 */
    const double step = ldexp(1.0, E - 3);
    double q = x / step; /* exact: step is a power of two */
    q = round_up ? ceil(q) : nearbyint(q);
    const double v = q * step; /* <= 448: 448 is a grid point */
    if (v < ldexp(1.0, -6)) return (uint8_t)q; /* subnormal (or zero) */
    int ev;
    frexp(v, &ev);
    const int Ev = ev - 1;
    const int m = (int)((v / ldexp(1.0, Ev) - 1.0) * 8.0);
    return (uint8_t)(((Ev + 7) << 3) | m);
}

double kvo_fp16_to_double(uint16_t h) {
    const int e = (h >> 10) & 31, m = h & 1023;
    const double mag = e == 0 ? ldexp((double)m, -24) : ldexp(1.0 + m / 1024.0, e - 15);
    return (h & 0x8000) ? -mag : mag;
}

uint16_t kvo_fp16_from_double(double x) {
    const uint16_t sign = x < 0.0 ? 0x8000 : 0;
    const double ax = fabs(x);
    if (ax >= 65504.0) return sign | 0x7BFF;
    if (ax == 0.0) return sign;
    int ex;
    frexp(ax, &ex);
    int E = ex - 1;
    if (E < -14) E = -14;
    const double step = ldexp(1.0, E - 10);
    const double v = nearbyint(ax / step) * step;
    if (v < ldexp(1.0, -14)) return sign | (uint16_t)(v / ldexp(1.0, -24));
    int ev;
    frexp(v, &ev);
    const int Ev = ev - 1;
    const int m = (int)((v / ldexp(1.0, Ev) - 1.0) * 1024.0);
    return sign | (uint16_t)(((Ev + 15) << 10) | m);
}

/* ------------------------------------------------------------------------------------------
 * Hadamard rotation (Sec. 2.2, Sec. 3.3, App. A).  Sylvester-ordered Walsh-Hadamard matrix
 * H[i][j] = (-1)^popcount(i & j) / sqrt(128): symmetric, orthonormal and its own inverse.
 * Computed with the textbook in-place butterflies, stride 1, 2, 4, ..., 64.
 * ------------------------------------------------------------------------------------------ */
void kvo_hadamard128(double *x) {
    for (int h = 1; h < D; h <<= 1) {
        for (int i = 0; i < D; i += 2 * h) {
            for (int j = i; j < i + h; ++j) {
                double a = x[j], b = x[j + h];
                x[j] = a + b;
                x[j + h] = a - b;
            }
        }
    }
    const double s = 1.0 / sqrt((double)D);
    for (int i = 0; i < D; ++i) x[i] *= s;
}

/* ------------------------------------------------------------------------------------------
 * VarN (Sec. 3.3, App. H, Algorithm 1) on one tile T of R rows and C columns, row-major; rows
 * are the tile's tokens, columns its channels.
 *
 * The method looks for a row scale S_r and a column scale S_c such that the balanced tile
 * T[r][c] / (S_c[c] S_r[r]) has lines of equal spread along both axes.  The scales are kept as
 * logarithms L_c, L_r (zero at the start).  One iteration balances the columns and then the
 * rows (the column scales come first, reading A1): a line's variance v in the current balanced
 * tile is clamped to [c_min, c_max] and the line's log-scale moves by log(sqrt(v)), i.e. by half
 * of log v, then is clamped to [log_lo, log_hi].  Dividing the line by sqrt(v) gives it unit
 * variance, so without the clamps every line of the axis just balanced has variance exactly 1.
 * After both axes the imbalance Imb of the current tile is measured (the ratio of the largest
 * to the smallest line variance of each axis, summed over the two axes, the smallest floored
 * at imb_floor), and the scales of the best state seen so far are kept; the start state counts
 * as iteration 0 and a later iteration displaces an earlier one of equal Imb.
 * ------------------------------------------------------------------------------------------ */

enum { AXIS_COLUMNS = 0, AXIS_ROWS = 1 };

/* Two-pass (mean-centred) variance of n values spaced `stride` apart, divisor n - ddof. */
static double variance(const double *v, int n, int stride, int ddof) {
    double mean = 0.0;
    for (int i = 0; i < n; ++i) mean += v[(size_t)i * stride];
    mean /= (double)n;
    double ss = 0.0;
    for (int i = 0; i < n; ++i) {
        double d = v[(size_t)i * stride] - mean;
        ss += d * d;
    }
    return ss / (double)(n - ddof);
}

/* Variance of line i of the axis: column i taken over the R rows, or row i over the C columns. */
static double line_variance(const double *X, int R, int C, int axis, int i, int ddof) {
    return axis == AXIS_COLUMNS ? variance(X + i, R, C, ddof) : variance(X + (size_t)i * C, C, 1, ddof);
}

static double clampd(double x, double lo, double hi) { return x < lo ? lo : (x > hi ? hi : x); }

/* Largest over smallest line variance of one axis (the smallest floored); 1 when balanced. */
static double spread_ratio(const double *X, int R, int C, int axis, int ddof, double floor_) {
    const int n = axis == AXIS_COLUMNS ? C : R;
    double vmax = -INFINITY, vmin = INFINITY;
    for (int i = 0; i < n; ++i) {
        const double v = line_variance(X, R, C, axis, i, ddof);
        vmax = fmax(vmax, v);
        vmin = fmin(vmin, v);
    }
    return vmax / fmax(vmin, floor_);
}

/* Imb(X) of Algorithm 1: the spread ratio of the rows plus that of the columns. */
double kvo_imbalance(const double *X, int R, int C, int ddof, double floor_) {
    return spread_ratio(X, R, C, AXIS_ROWS, ddof, floor_) + spread_ratio(X, R, C, AXIS_COLUMNS, ddof, floor_);
}

/* The tile and its current log-scales. */
typedef struct {
    const double *T;
    int R, C;
    double *Lc, *Lr; /* log-scale of every column and of every row */
    double *Cur;     /* current balanced tile */
} varn_state;

/* Cur[r][c] = T[r][c] divided by e^{Lc[c]}, and the quotient divided by e^{Lr[r]}. */
static void rebalance(varn_state *s) {
    for (int r = 0; r < s->R; ++r)
        for (int c = 0; c < s->C; ++c)
            s->Cur[(size_t)r * s->C + c] = (s->T[(size_t)r * s->C + c] / exp(s->Lc[c])) / exp(s->Lr[r]);
}

/* One half-iteration: every line of the axis takes half the log of its clamped variance into
 * its log-scale (clamped), measured on the tile before any of them moves; then Cur is redone. */
static void balance_axis(varn_state *s, int axis, const kvo_params *p) {
    const int n = axis == AXIS_COLUMNS ? s->C : s->R;
    double *L = axis == AXIS_COLUMNS ? s->Lc : s->Lr;
    for (int i = 0; i < n; ++i) {
        const double v = clampd(line_variance(s->Cur, s->R, s->C, axis, i, p->ddof), p->c_min, p->c_max);
        L[i] = clampd(L[i] + 0.5 * log(v), p->log_lo, p->log_hi);
    }
    rebalance(s);
}

/* The scales of the best state so far: S_c*, S_r* (linear), its Imb and iteration. */
typedef struct {
    double *Sc, *Sr;
    double I;
    int k;
} varn_best;

/* Keep iteration k's scales if its imbalance I is no larger than the best so far (the later
 * one wins a tie), or, with force_best >= 0, exactly when k is that iteration (test use). */
static void keep_if_best(varn_best *b, const varn_state *s, double I, int k, const kvo_params *p) {
    const int take = k == 0 || (p->force_best >= 0 ? k == p->force_best : I <= b->I);
    if (!take) return;
    b->I = I;
    b->k = k;
    for (int c = 0; c < s->C; ++c) b->Sc[c] = exp(s->Lc[c]);
    for (int r = 0; r < s->R; ++r) b->Sr[r] = exp(s->Lr[r]);
}

/*
 * VarN on one tile.
 *   T[R*C] (row-major) in; Sc[C], Sr[R] out: the kept scales S_c*, S_r*;
 *   Bal[R*C] out (optional): T with column c divided by Sc[c], then row r by Sr[r].
 * Optional histories, indexed by iteration k = 0..K (0 = the start state):
 *   imb_hist[K+1], Lc_hist[(K+1)*C], Lr_hist[(K+1)*R].
 * *best_iter (optional) receives the iteration whose scales were kept.
 */
void kvo_varn(const double *T, int R, int C, const kvo_params *p, double *Sc, double *Sr, double *Bal,
              double *imb_hist, double *Lc_hist, double *Lr_hist, int *best_iter) {
    varn_state s = {T, R, C, calloc((size_t)C, sizeof(double)), calloc((size_t)R, sizeof(double)),
                    malloc((size_t)R * C * sizeof(double))};
    varn_best best = {Sc, Sr, INFINITY, -1};
    rebalance(&s);
    for (int k = 0; k <= p->varn_iters; ++k) {
        if (k > 0) {
            balance_axis(&s, AXIS_COLUMNS, p);
            balance_axis(&s, AXIS_ROWS, p);
        }
        const double I = kvo_imbalance(s.Cur, R, C, p->ddof, p->imb_floor);
        keep_if_best(&best, &s, I, k, p);
        if (imb_hist) imb_hist[k] = I;
        if (Lc_hist) memcpy(Lc_hist + (size_t)k * C, s.Lc, (size_t)C * sizeof(double));
        if (Lr_hist) memcpy(Lr_hist + (size_t)k * R, s.Lr, (size_t)R * sizeof(double));
    }
    if (Bal)
        for (int r = 0; r < R; ++r)
            for (int c = 0; c < C; ++c) Bal[(size_t)r * C + c] = (T[(size_t)r * C + c] / Sc[c]) / Sr[r];
    if (best_iter) *best_iter = best.k;
    free(s.Lc);
    free(s.Lr);
    free(s.Cur);
}

/* ------------------------------------------------------------------------------------------
 * Asymmetric round-to-nearest over one group of n values (Sec. 2.1, Eq. 1):
 *   mn = min, mx = max, s = (mx - mn) / (2^bits - 1)   (s := 1 when mx == mn)
 *   u = (x - mn) / s, code = clamp(round-half-even(u), 0, 2^bits - 1)
 * The quotient u is evaluated as (2^bits - 1)(x - mn) / (mx - mn), the same real number with a
 * single rounding at the end, so a value that lies exactly halfway between two levels gives an
 * exact half-integer u and is rounded half to even.  Eq. 1 writes the dequantized value as
 * (code + z) * s with z = mn / s; the stored form here is the equivalent code * s + mn.
 * u_out (optional) receives the unrounded quotients.
 * ------------------------------------------------------------------------------------------ */
void kvo_rtn_group(const double *x, int n, int stride, int bits, uint8_t *codes, int code_stride,
                   double *mn_out, double *s_out, double *u_out, int u_stride) {
    double mn = INFINITY, mx = -INFINITY;
    for (int i = 0; i < n; ++i) {
        mn = fmin(mn, x[(size_t)i * stride]);
        mx = fmax(mx, x[(size_t)i * stride]);
    }
    const double qmax = (double)((1 << bits) - 1);
    const double range = mx - mn;
    for (int i = 0; i < n; ++i) {
        const double d = x[(size_t)i * stride] - mn;
        double u = range > 0.0 ? (qmax * d) / range : d; /* d = 0 for a constant group */
        double q = nearbyint(u); /* default rounding mode: to nearest, ties to even */
        if (q < 0.0) q = 0.0;
        if (q > qmax) q = qmax;
        codes[(size_t)i * code_stride] = (uint8_t)q;
        if (u_out) u_out[(size_t)i * u_stride] = u;
    }
    *mn_out = mn;
    *s_out = range > 0.0 ? range / qmax : 1.0;
}

/* ------------------------------------------------------------------------------------------
 * Quantize one 128-token x 128-channel tile X (token-major) of K or V (Fig. 2, Sec. 3.3):
 *   1. T[t,:] = H X[t,:]                     Hadamard along head_dim, per token
 *   2. (B, S_c*, S_r*) = VarN(T)             Algorithm 1, rows = tokens, columns = channels
 *   3. RTN on B along the group axis         keys: per channel over the 128 tokens,
 *                                            values: per token over the 128 channels (Sec. 2.1)
 *   4. absorb the Sinkhorn scale of the group axis into the RTN scale and offset (App. D):
 *        keys:   a[c] = s_c * S_c*[c],  b[c] = mn_c * S_c*[c],  s2[t] = S_r*[t]
 *        values: a[t] = s_t * S_r*[t],  b[t] = mn_t * S_r*[t],  s2[c] = S_c*[c]
 *      so that the dequantized rotated tile is  (code * a + b) * s2.
 * Outputs: codes[128*128] token-major; a, b, s2 rounded to fp32.
 *
 * Compact aux (p->aux == 1): the stored values are narrow, so they are rounded first and the
 * codes are computed against the stored values ("absorb, then round"):
 *   s2  = E4M3 nearest of 2^e times the other-axis scale (kept within [2^-6, 448]);
 *   z   = T / s2 along the other axis (= B times the group-axis Sinkhorn scale, over 2^e: RTN
 *         of a group does not depend on a common factor, so that scale is absorbed exactly);
 *   per group: mn, mx of z, step = (mx - mn) / (2^bits - 1) (1 when mx == mn),
 *   a   = E4M3 of step rounded upward (so [b, b + qmax * a] covers the group), b = binary16
 *         nearest of mn, u = (z - b) / a, code = clamp(round-half-even(u), 0, qmax).
 *   e   = a tile-wide power of two moved from a and b into s2 (App. D stores both scales in
 *         FP8 but does not say how the magnitude is split; both are E4M3, at most 448, while
 *         their product is fixed by the data): the smallest e >= 0 for which the largest step
 *         of the tile is at most 448, taken no further than the largest other-axis scale
 *         times 2^e stays within 448, and only when no other-axis scale lies below 2^-6
 *         (the clamp of s2; with Algorithm 1's log clamp at -0.3 none does).  Without it a key
 *         tile of magnitude ~100 with outlier channels saturates a at 448 and its range no
 *         longer covers the group.
 * The dequantized value (code * a + b) * s2 then keeps the RTN error bound a * s2 / 2 (plus the
 * rounding of b).
 * Optional debug outputs (NULL to skip): T_out[128*128], Bal_out[128*128], u_out[128*128]
 * (token-major unrounded quotients), Sc_out[128], Sr_out[128], imb_hist[K+1], best_iter,
 * pre_out[3*128]: a, b, s2 before their rounding to the stored format.
 * ------------------------------------------------------------------------------------------ */
/* Stored (E4M3) other-axis scale for a tile-wide shift 2^e. */
static double stored_s2(double so, int e) {
    return kvo_e4m3_to_double(kvo_e4m3_from_double(clampd(ldexp(so, e), ldexp(1.0, -6), 448.0), 0));
}

/* Largest group step (mx - mn) / qmax of z = T / s2 over the tile, for the shift 2^e. */
static double largest_step(const double *T, const double *So, int e, int kind, double qmax) {
    double best = 0.0;
    for (int g = 0; g < 128; ++g) {
        double mn = INFINITY, mx = -INFINITY;
        for (int i = 0; i < 128; ++i) {
            const double x = kind == KVO_KEYS ? T[(size_t)i * D + g] : T[(size_t)g * D + i];
            const double z = x / stored_s2(So[i], e);
            mn = fmin(mn, z);
            mx = fmax(mx, z);
        }
        best = fmax(best, (mx - mn) / qmax);
    }
    return best;
}

static void quantize_compact(const double *T, const double *Sc, const double *Sr, int kind, int bits,
                             uint8_t *codes, float *a, float *b, float *s2, double *u_out, double *pre_out) {
    const double qmax = (double)((1 << bits) - 1);
    const double *So = kind == KVO_KEYS ? Sr : Sc; /* other-axis scale: per token for keys */
    double so_max = 0.0, so_min = INFINITY;
    for (int i = 0; i < 128; ++i) {
        so_max = fmax(so_max, So[i]);
        so_min = fmin(so_min, So[i]);
    }
    int e = 0;
    if (so_min >= ldexp(1.0, -6))
        while (largest_step(T, So, e, kind, qmax) > 448.0 && ldexp(so_max, e + 1) <= 448.0) ++e;
    double s2q[128];
    for (int i = 0; i < 128; ++i) {
        s2q[i] = stored_s2(So[i], e);
        s2[i] = (float)s2q[i];
        if (pre_out) pre_out[256 + i] = ldexp(So[i], e);
    }
    double z[128];
    for (int g = 0; g < 128; ++g) { /* group: channel g (keys) or token g (values) */
        double mn = INFINITY, mx = -INFINITY;
        for (int i = 0; i < 128; ++i) { /* i: token (keys) or channel (values) */
            const double x = kind == KVO_KEYS ? T[(size_t)i * D + g] : T[(size_t)g * D + i];
            z[i] = x / s2q[i];
            mn = fmin(mn, z[i]);
            mx = fmax(mx, z[i]);
        }
        double step = (mx - mn) / qmax;
        if (step == 0.0) step = 1.0;
        const double aq = kvo_e4m3_to_double(kvo_e4m3_from_double(step, 1));
        const double bq = kvo_fp16_to_double(kvo_fp16_from_double(mn));
        a[g] = (float)aq;
        b[g] = (float)bq;
        if (pre_out) {
            pre_out[g] = step;
            pre_out[128 + g] = mn;
        }
        for (int i = 0; i < 128; ++i) {
            const double u = (z[i] - bq) / aq;
            double q = nearbyint(u);
            if (q < 0.0) q = 0.0;
            if (q > qmax) q = qmax;
            const size_t at = kind == KVO_KEYS ? (size_t)i * D + g : (size_t)g * D + i;
            codes[at] = (uint8_t)q;
            if (u_out) u_out[at] = u;
        }
    }
}

void kvo_quantize_tile(const double *X, int kind, const kvo_params *p, uint8_t *codes, float *a, float *b,
                       float *s2, double *T_out, double *Bal_out, double *u_out, double *Sc_out, double *Sr_out,
                       double *imb_hist, int *best_iter, double *pre_out) {
    double *T = malloc((size_t)G * D * sizeof(double));
    double *Bal = malloc((size_t)G * D * sizeof(double));
    double Sc[D], Sr[G];
    memcpy(T, X, (size_t)G * D * sizeof(double));
    if (p->rotate)
        for (int t = 0; t < G; ++t) kvo_hadamard128(T + (size_t)t * D);
    kvo_varn(T, G, D, p, Sc, Sr, Bal, imb_hist, NULL, NULL, best_iter);

    if (p->aux == 1) {
        quantize_compact(T, Sc, Sr, kind, p->bits, codes, a, b, s2, u_out, pre_out);
    } else if (kind == KVO_KEYS) {
        for (int c = 0; c < D; ++c) {
            double mn, s;
            kvo_rtn_group(Bal + c, G, D, p->bits, codes + c, D, &mn, &s, u_out ? u_out + c : NULL, D);
            a[c] = (float)(s * Sc[c]);
            b[c] = (float)(mn * Sc[c]);
        }
        for (int t = 0; t < G; ++t) s2[t] = (float)Sr[t];
    } else {
        for (int t = 0; t < G; ++t) {
            double mn, s;
            kvo_rtn_group(Bal + (size_t)t * D, D, 1, p->bits, codes + (size_t)t * D, 1, &mn, &s,
                          u_out ? u_out + (size_t)t * D : NULL, 1);
            a[t] = (float)(s * Sr[t]);
            b[t] = (float)(mn * Sr[t]);
        }
        for (int c = 0; c < D; ++c) s2[c] = (float)Sc[c];
    }
    if (T_out) memcpy(T_out, T, (size_t)G * D * sizeof(double));
    if (Bal_out) memcpy(Bal_out, Bal, (size_t)G * D * sizeof(double));
    if (Sc_out) memcpy(Sc_out, Sc, sizeof Sc);
    if (Sr_out) memcpy(Sr_out, Sr, sizeof Sr);
    free(T);
    free(Bal);
}

/* ------------------------------------------------------------------------------------------
 * Packed tile format (this library's own storage format; the paper fixes only what is
 * stored per group, App. D).  A tile is
 *     codes region: bits * 2048 bytes (128 x 128 codes of `bits` bits)
 *     aux 0: a[128], b[128], s2[128]: little-endian binary32, in index order (token or channel)
 *     aux 1: b[128] little-endian binary16, then a[128] and s2[128] as E4M3 bytes
 * Codes are grouped in "units" of 16 codes; a unit is bits/2 consecutive 32-bit
 * little-endian words.  Write unit u as u = 512*sigma + 8*L + w (sigma in 0..1, L in 0..63,
 * w in 0..7) and p = 8/bits; unit u starts at word
 *     512*(bits/2)*sigma + 256*(w / p) + 4*L + (bits/2)*(w % p).
 * Inside a unit, code number e = 4*s + q (s, q in 0..3) sits in word  s / p  at bit
 * 8*q + bits*(s % p).  The unit index and e of code (t, c) are, with sigma = t / 64:
 *   keys:   unit = (sigma*64 + 16*((c % 64) / 16) + t % 16) * 8 + 2*((t % 64) / 16) + c / 64,
 *           e = c % 16
 *   values: unit = (sigma*64 + 16*((t % 16) / 4) + c % 16) * 8 + c / 16,
 *           e = 4*((t % 64) / 16) + t % 4
 * ------------------------------------------------------------------------------------------ */
size_t kvo_tile_bytes(int bits, int aux) { return (size_t)bits * 2048 + (aux == 1 ? 512 : 3 * 128 * 4); }

static void code_location(int kind, int bits, int t, int c, size_t *word, int *shift) {
    int sigma = t / 64;
    size_t unit;
    int e;
    if (kind == KVO_KEYS) {
        unit = ((size_t)sigma * 64 + 16 * ((c % 64) / 16) + t % 16) * 8 + 2 * ((t % 64) / 16) + c / 64;
        e = c % 16;
    } else {
        unit = ((size_t)sigma * 64 + 16 * ((t % 16) / 4) + c % 16) * 8 + c / 16;
        e = 4 * ((t % 64) / 16) + t % 4;
    }
    int s = e / 4, q = e % 4, per = 8 / bits;
    size_t wpu = (size_t)(bits / 2), sg = unit / 512, L = (unit / 8) % 64, w = unit % 8;
    size_t start = 512 * wpu * sg + 256 * (w / (size_t)per) + 4 * L + wpu * (w % (size_t)per);
    *word = start + (size_t)(s / per);
    *shift = 8 * q + bits * (s % per);
}

static void put_f32(uint8_t *dst, float v) { memcpy(dst, &v, 4); } /* host is little-endian */
static float get_f32(const uint8_t *src) { float v; memcpy(&v, src, 4); return v; }

void kvo_pack_tile(const uint8_t *codes, const float *a, const float *b, const float *s2, int kind, int bits,
                   int aux, uint8_t *dst) {
    size_t ncode_bytes = (size_t)bits * 2048;
    uint32_t *words = calloc(ncode_bytes / 4, sizeof(uint32_t));
    for (int t = 0; t < G; ++t)
        for (int c = 0; c < D; ++c) {
            size_t w;
            int sh;
            code_location(kind, bits, t, c, &w, &sh);
            words[w] |= (uint32_t)codes[(size_t)t * D + c] << sh;
        }
    for (size_t w = 0; w < ncode_bytes / 4; ++w) { /* little-endian words */
        dst[4 * w + 0] = (uint8_t)(words[w]);
        dst[4 * w + 1] = (uint8_t)(words[w] >> 8);
        dst[4 * w + 2] = (uint8_t)(words[w] >> 16);
        dst[4 * w + 3] = (uint8_t)(words[w] >> 24);
    }
    for (int i = 0; i < 128; ++i) {
        if (aux == 1) { /* the values are already on the narrow grids: exact re-encoding */
            const uint16_t h = kvo_fp16_from_double((double)b[i]);
            dst[ncode_bytes + 2 * i] = (uint8_t)h;
            dst[ncode_bytes + 2 * i + 1] = (uint8_t)(h >> 8);
            dst[ncode_bytes + 256 + i] = kvo_e4m3_from_double((double)a[i], 0);
            dst[ncode_bytes + 384 + i] = kvo_e4m3_from_double((double)s2[i], 0);
        } else {
            put_f32(dst + ncode_bytes + 4 * i, a[i]);
            put_f32(dst + ncode_bytes + 512 + 4 * i, b[i]);
            put_f32(dst + ncode_bytes + 1024 + 4 * i, s2[i]);
        }
    }
    free(words);
}

void kvo_unpack_tile(const uint8_t *src, int kind, int bits, int aux, uint8_t *codes, float *a, float *b,
                     float *s2) {
    size_t ncode_bytes = (size_t)bits * 2048;
    const uint32_t mask = (1u << bits) - 1u;
    for (int t = 0; t < G; ++t)
        for (int c = 0; c < D; ++c) {
            size_t w;
            int sh;
            code_location(kind, bits, t, c, &w, &sh);
            uint32_t word = (uint32_t)src[4 * w] | (uint32_t)src[4 * w + 1] << 8 | (uint32_t)src[4 * w + 2] << 16 |
                            (uint32_t)src[4 * w + 3] << 24;
            codes[(size_t)t * D + c] = (uint8_t)((word >> sh) & mask);
        }
    for (int i = 0; i < 128; ++i) {
        if (aux == 1) {
            const uint16_t h = (uint16_t)(src[ncode_bytes + 2 * i] | src[ncode_bytes + 2 * i + 1] << 8);
            if (b) b[i] = (float)kvo_fp16_to_double(h);
            if (a) a[i] = (float)kvo_e4m3_to_double(src[ncode_bytes + 256 + i]);
            if (s2) s2[i] = (float)kvo_e4m3_to_double(src[ncode_bytes + 384 + i]);
        } else {
            if (a) a[i] = get_f32(src + ncode_bytes + 4 * i);
            if (b) b[i] = get_f32(src + ncode_bytes + 512 + 4 * i);
            if (s2) s2[i] = get_f32(src + ncode_bytes + 1024 + 4 * i);
        }
    }
}

/*
 * Dequantize a packed tile back to the unrotated domain, in double:
 *   rotated: keys   Xr[t][c] = (code * a[c] + b[c]) * s2[t]
 *            values Xr[t][c] = (code * a[t] + b[t]) * s2[c]
 *   then X[t,:] = H Xr[t,:] (H is its own inverse).  Out: X[128*128] token-major.
 */
void kvo_dequantize_tile(const uint8_t *src, int kind, int bits, int aux, int rotate, double *X) {
    uint8_t *codes = malloc((size_t)G * D);
    float a[128], b[128], s2[128];
    kvo_unpack_tile(src, kind, bits, aux, codes, a, b, s2);
    for (int t = 0; t < G; ++t) {
        for (int c = 0; c < D; ++c) {
            double q = (double)codes[(size_t)t * D + c];
            X[(size_t)t * D + c] = kind == KVO_KEYS ? (q * (double)a[c] + (double)b[c]) * (double)s2[t]
                                                    : (q * (double)a[t] + (double)b[t]) * (double)s2[c];
        }
        if (rotate) kvo_hadamard128(X + (size_t)t * D);
    }
    free(codes);
}

/* Quantize + pack one tile whose input is fp32 (dtype 0) or bf16 (dtype 1) at `x` with the
 * given token stride (in elements; channels contiguous). */
void kvo_quantize_pack(const void *x, int dtype, int64_t token_stride, int kind, const kvo_params *p, uint8_t *dst) {
    double *X = malloc((size_t)G * D * sizeof(double));
    uint8_t *codes = malloc((size_t)G * D);
    float a[128], b[128], s2[128];
    for (int t = 0; t < G; ++t)
        for (int c = 0; c < D; ++c)
            X[(size_t)t * D + c] = dtype == 0 ? (double)((const float *)x)[t * token_stride + c]
                                              : kvo_bf16_to_double(((const uint16_t *)x)[t * token_stride + c]);
    kvo_quantize_tile(X, kind, p, codes, a, b, s2, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL);
    kvo_pack_tile(codes, a, b, s2, kind, p->bits, p->aux, dst);
    free(X);
    free(codes);
}

/*
 * Batched quantize: tile (i, j) reads x + i*x_outer + j*x_inner (elements) and writes the packed
 * tile to out + (i*out_outer + j*out_inner) * tile_bytes.  Tiles are independent; OpenMP
 * distributes them over the host's threads.
 */
void kvo_quantize_tiles(const void *x, int dtype, int64_t n_outer, int64_t n_inner, int64_t x_outer, int64_t x_inner,
                        int64_t token_stride, int kind, const kvo_params *p, uint8_t *out, int64_t out_outer,
                        int64_t out_inner) {
    const size_t tb = kvo_tile_bytes(p->bits, p->aux);
    const size_t esz = dtype == 0 ? 4 : 2;
#pragma omp parallel for collapse(2) schedule(dynamic)
    for (int64_t i = 0; i < n_outer; ++i)
        for (int64_t j = 0; j < n_inner; ++j)
            kvo_quantize_pack((const uint8_t *)x + (size_t)(i * x_outer + j * x_inner) * esz, dtype, token_stride,
                              kind, p, out + (size_t)(i * out_outer + j * out_inner) * tb);
}

/* ------------------------------------------------------------------------------------------
 * Cache regions (App. D "Quantization"): the first n_sink tokens of a sequence stay in bf16
 * (sink), then come full groups of 128 quantized tokens (body), then the most recent
 * (len - n_sink) % 128 tokens in bf16 (residual).  Residual and sink hold the tokens as given
 * (unrotated); body tiles are stored in the rotated domain and un-rotated on dequantization.
 *
 * Host layout shared with the GPU library (described in its header, re-derived here):
 *   k_body, v_body:   [batch][n_kv][max_blocks] packed tiles
 *   k_resid, v_resid: [batch][n_kv][128][128] bf16
 *   k_sink, v_sink:   [batch][n_kv][n_sink][128] bf16 (unused when n_sink == 0)
 *   seq_len:          [batch] int32
 * ------------------------------------------------------------------------------------------ */
typedef struct {
    int32_t batch, n_kv, max_blocks, n_sink, bits, aux, rotate;
    uint8_t *k_body, *v_body;
    uint16_t *k_resid, *v_resid, *k_sink, *v_sink;
    int32_t *seq_len;
    const int32_t *block_table; /* NULL: dense body; else [batch][max_blocks] pool block ids and
                                   bodies [n_phys][n_kv] tiles (the paged layout) */
    int32_t n_phys;
} kvo_cache;

/* Body tile blk of (sequence b, kv head kh): dense [batch][n_kv][max_blocks] or, paged, tile kh
 * of pool block block_table[b][blk].  NULL for a pool id outside [0, n_phys). */
static uint8_t *body_tile(const kvo_cache *cc, uint8_t *body, int32_t b, int32_t kh, int32_t blk) {
    const size_t tb = kvo_tile_bytes(cc->bits, cc->aux);
    if (!cc->block_table) return body + (((size_t)b * cc->n_kv + kh) * cc->max_blocks + blk) * tb;
    const int32_t id = cc->block_table[(size_t)b * cc->max_blocks + blk];
    if (id < 0 || id >= cc->n_phys) return NULL;
    return body + ((size_t)id * cc->n_kv + kh) * tb;
}

static void region_sizes(const kvo_cache *cc, int32_t len, int32_t *n_sink_used, int32_t *n_blocks, int32_t *n_resid) {
    if (len <= cc->n_sink) {
        *n_sink_used = len;
        *n_blocks = 0;
        *n_resid = 0;
    } else {
        *n_sink_used = cc->n_sink;
        *n_blocks = (len - cc->n_sink) / G;
        *n_resid = (len - cc->n_sink) % G;
    }
}

/*
 * Gather the full-precision view of one (sequence, kv-head) stream: keys and values of all
 * `len` tokens in the unrotated domain, in token order (sink, body, residual).
 * K, V: [len][128] doubles, caller-allocated.
 */
void kvo_gather_stream(const kvo_cache *cc, int32_t bi, int32_t kh, double *K, double *V) {
    const int32_t len = cc->seq_len[bi];
    int32_t ns, nb, nr;
    region_sizes(cc, len, &ns, &nb, &nr);
    const size_t stream = (size_t)bi * cc->n_kv + kh;
    int32_t t = 0;
    for (int32_t i = 0; i < ns; ++i, ++t)
        for (int c = 0; c < D; ++c) {
            K[(size_t)t * D + c] = kvo_bf16_to_double(cc->k_sink[(stream * cc->n_sink + i) * D + c]);
            V[(size_t)t * D + c] = kvo_bf16_to_double(cc->v_sink[(stream * cc->n_sink + i) * D + c]);
        }
    for (int32_t blk = 0; blk < nb; ++blk, t += G) {
        kvo_dequantize_tile(body_tile(cc, cc->k_body, bi, kh, blk), KVO_KEYS, cc->bits, cc->aux, cc->rotate,
                            K + (size_t)t * D);
        kvo_dequantize_tile(body_tile(cc, cc->v_body, bi, kh, blk), KVO_VALUES, cc->bits, cc->aux, cc->rotate,
                            V + (size_t)t * D);
    }
    for (int32_t i = 0; i < nr; ++i, ++t)
        for (int c = 0; c < D; ++c) {
            K[(size_t)t * D + c] = kvo_bf16_to_double(cc->k_resid[(stream * G + i) * D + c]);
            V[(size_t)t * D + c] = kvo_bf16_to_double(cc->v_resid[(stream * G + i) * D + c]);
        }
}

/* Plain attention of one query over n tokens: o = softmax(scale * K q) V, max-subtracted. */
void kvo_attend(const double *q, const double *K, const double *V, int32_t n, double scale, double *o) {
    double *s = malloc((size_t)(n > 0 ? n : 1) * sizeof(double));
    double m = -INFINITY;
    for (int32_t t = 0; t < n; ++t) {
        double acc = 0.0;
        for (int c = 0; c < D; ++c) acc += q[c] * K[(size_t)t * D + c];
        s[t] = scale * acc;
        m = fmax(m, s[t]);
    }
    double l = 0.0;
    for (int c = 0; c < D; ++c) o[c] = 0.0;
    for (int32_t t = 0; t < n; ++t) {
        double pt = exp(s[t] - m);
        l += pt;
        for (int c = 0; c < D; ++c) o[c] += pt * V[(size_t)t * D + c];
    }
    for (int c = 0; c < D; ++c) o[c] = n > 0 ? o[c] / l : 0.0;
    free(s);
}

/*
 * Decode attention over the whole cache: for sequence b and query head h (kv head
 * h / (n_q / n_kv)), out[b][h][:] = softmax(scale * q . K^T) V over every cached token.
 * q: [batch][n_q][128] as fp32 (dtype 0) or bf16 (dtype 1); out: [batch][n_q][128] doubles.
 */
void kvo_decode(const kvo_cache *cc, int32_t n_q, const void *q, int dtype, double scale, double *out) {
    const int32_t grp = n_q / cc->n_kv;
#pragma omp parallel for collapse(2) schedule(dynamic)
    for (int32_t bi = 0; bi < cc->batch; ++bi)
        for (int32_t kh = 0; kh < cc->n_kv; ++kh) {
            const int32_t len = cc->seq_len[bi];
            double *K = malloc((size_t)(len > 0 ? len : 1) * D * sizeof(double));
            double *V = malloc((size_t)(len > 0 ? len : 1) * D * sizeof(double));
            kvo_gather_stream(cc, bi, kh, K, V);
            for (int32_t j = 0; j < grp; ++j) {
                int32_t h = kh * grp + j;
                double qd[D];
                size_t qoff = ((size_t)bi * n_q + h) * D;
                for (int c = 0; c < D; ++c)
                    qd[c] = dtype == 0 ? (double)((const float *)q)[qoff + c]
                                       : kvo_bf16_to_double(((const uint16_t *)q)[qoff + c]);
                kvo_attend(qd, K, V, len, scale, out + qoff);
            }
            free(K);
            free(V);
        }
}

/*
 * Append one token per (sequence, kv head) (the streaming write of Fig. 4's pseudo-decode and
 * App. D's three regions): k_new, v_new are [batch][n_kv][128] bf16.  The token goes to the
 * sink while the sequence is shorter than n_sink, otherwise to the residual; when the
 * residual reaches 128 tokens it is quantized (keys and values) into the next body tile and
 * emptied.  Returns 0, or -3 if a sequence has no free body slot for the flush.
 */
int kvo_append(kvo_cache *cc, const uint16_t *k_new, const uint16_t *v_new, const kvo_params *p) {
    if (p->bits != cc->bits || p->aux != cc->aux || p->rotate != cc->rotate) return -1;
    for (int32_t bi = 0; bi < cc->batch; ++bi) {
        int32_t len = cc->seq_len[bi];
        int32_t ns, nb, nr;
        region_sizes(cc, len, &ns, &nb, &nr);
        if (len >= cc->n_sink && nr == G - 1 && nb >= cc->max_blocks) return -3;
    }
    for (int32_t bi = 0; bi < cc->batch; ++bi) {
        int32_t len = cc->seq_len[bi];
        int32_t ns, nb, nr;
        region_sizes(cc, len, &ns, &nb, &nr);
        for (int32_t kh = 0; kh < cc->n_kv; ++kh) {
            const size_t stream = (size_t)bi * cc->n_kv + kh;
            const uint16_t *kn = k_new + stream * D, *vn = v_new + stream * D;
            if (len < cc->n_sink) {
                memcpy(cc->k_sink + (stream * cc->n_sink + len) * D, kn, D * 2);
                memcpy(cc->v_sink + (stream * cc->n_sink + len) * D, vn, D * 2);
                continue;
            }
            memcpy(cc->k_resid + (stream * G + nr) * D, kn, D * 2);
            memcpy(cc->v_resid + (stream * G + nr) * D, vn, D * 2);
            if (nr + 1 == G) {
                uint8_t *kt = body_tile(cc, cc->k_body, bi, kh, nb), *vt = body_tile(cc, cc->v_body, bi, kh, nb);
                if (!kt || !vt) return -4;
                kvo_quantize_pack(cc->k_resid + stream * G * D, 1, D, KVO_KEYS, p, kt);
                kvo_quantize_pack(cc->v_resid + stream * G * D, 1, D, KVO_VALUES, p, vt);
            }
        }
        cc->seq_len[bi] = len + 1;
    }
    return 0;
}

/* ------------------------------------------------------------------------------------------
 * Error decomposition of Sec. 3.1, Eq. 3, per token (row of 128): with the angle theta
 * between k and its dequantized k_dq,
 *   E_T = |k - k_dq|^2                         total error
 *   E_M = (|k| - |k_dq|)^2                     magnitude error
 *   E_D = 2 |k| |k_dq| (1 - cos theta)         directional error,   E_T = E_M + E_D.
 * E_D is formed as 2 (|k| |k_dq| - k . k_dq), the same quantity without the angle.
 * ------------------------------------------------------------------------------------------ */
void kvo_error_decomposition(const double *K, const double *Kdq, int32_t n, double *ET, double *EM, double *ED) {
    for (int32_t t = 0; t < n; ++t) {
        const double *k = K + (size_t)t * D, *q = Kdq + (size_t)t * D;
        double kk = 0.0, qq = 0.0, kq = 0.0, e = 0.0;
        for (int c = 0; c < D; ++c) {
            kk += k[c] * k[c];
            qq += q[c] * q[c];
            kq += k[c] * q[c];
            e += (k[c] - q[c]) * (k[c] - q[c]);
        }
        const double nk = sqrt(kk), nq = sqrt(qq);
        ET[t] = e;
        EM[t] = (nk - nq) * (nk - nq);
        ED[t] = 2.0 * (nk * nq - kq);
    }
}

/*
 * Prefill whole prompts (the bulk counterpart of appending them token by token): k, v are
 * [total][n_kv][128] fp32 (dtype 0) or bf16 (dtype 1); sequence b owns rows cu[b] .. cu[b+1]-1.
 * Its cache becomes: seq_len = L, the first min(L, n_sink) tokens in the sink (bf16), each full
 * 128-token group after them quantized into body tiles 0, 1, ..., the remaining tokens in the
 * residual (bf16).  A sequence with L > max_len or more groups than max_blocks is not written
 * (seq_len 0) and the call returns -3; a bad pool id returns -4.
 */
int kvo_prefill(kvo_cache *cc, const void *k, const void *v, int dtype, const int32_t *cu, int32_t max_len,
                const kvo_params *p) {
    int too_long = 0, bad_id = 0;
    /* (sequence, kv head) streams are independent; OpenMP spreads them over the host's threads */
#pragma omp parallel for collapse(2) schedule(dynamic) reduction(|| : too_long, bad_id)
    for (int32_t bi = 0; bi < cc->batch; ++bi)
        for (int32_t kh = 0; kh < cc->n_kv; ++kh) {
            const int32_t L = cu[bi + 1] - cu[bi];
            int32_t ns, nb, nr;
            region_sizes(cc, L, &ns, &nb, &nr);
            if (L < 0 || L > max_len || nb > cc->max_blocks) {
                too_long = 1;
                continue;
            }
            const size_t stream = (size_t)bi * cc->n_kv + kh;
            for (int32_t t = 0; t < ns + nr; ++t) { /* sink rows, then residual rows */
                const int32_t row = t < ns ? t : L - nr + (t - ns);
                const size_t at = ((size_t)(cu[bi] + row) * cc->n_kv + kh) * D;
                uint16_t *kd = t < ns ? cc->k_sink + (stream * cc->n_sink + t) * D : cc->k_resid + (stream * G + t - ns) * D;
                uint16_t *vd = t < ns ? cc->v_sink + (stream * cc->n_sink + t) * D : cc->v_resid + (stream * G + t - ns) * D;
                for (int c = 0; c < D; ++c) {
                    kd[c] = dtype == 0 ? kvo_double_to_bf16(((const float *)k)[at + c]) : ((const uint16_t *)k)[at + c];
                    vd[c] = dtype == 0 ? kvo_double_to_bf16(((const float *)v)[at + c]) : ((const uint16_t *)v)[at + c];
                }
            }
            const size_t esz = dtype == 0 ? 4 : 2;
            for (int32_t blk = 0; blk < nb; ++blk) {
                uint8_t *kt = body_tile(cc, cc->k_body, bi, kh, blk), *vt = body_tile(cc, cc->v_body, bi, kh, blk);
                if (!kt || !vt) {
                    bad_id = 1;
                    continue;
                }
                const size_t at = ((size_t)(cu[bi] + ns + blk * G) * cc->n_kv + kh) * D;
                kvo_quantize_pack((const uint8_t *)k + at * esz, dtype, (int64_t)cc->n_kv * D, KVO_KEYS, p, kt);
                kvo_quantize_pack((const uint8_t *)v + at * esz, dtype, (int64_t)cc->n_kv * D, KVO_VALUES, p, vt);
            }
        }
    for (int32_t bi = 0; bi < cc->batch; ++bi) {
        const int32_t L = cu[bi + 1] - cu[bi];
        int32_t ns, nb, nr;
        region_sizes(cc, L, &ns, &nb, &nr);
        cc->seq_len[bi] = (L < 0 || L > max_len || nb > cc->max_blocks) ? 0 : L;
    }
    return bad_id ? -4 : (too_long ? -3 : 0);
}

/* Thread count of the parallel loops over tiles and streams (timing only; results do not
 * depend on it: every tile and stream is computed by one thread in a fixed order). */
void kvo_set_threads(int n) {
#ifdef _OPENMP
    omp_set_num_threads(n > 0 ? n : 1);
#else
    (void)n;
#endif
}
