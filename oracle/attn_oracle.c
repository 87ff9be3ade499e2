/*
 * CPU oracle for softmax attention and Rowmax-H15 attention.
 *
 * TEST INFRASTRUCTURE, NOT PRODUCT CODE.  Only the test suite, the smoke check
 * and the CPU-baseline leg of the benchmark may load this library.  It shares
 * no code, header, table or constant with the GPU library: everything below is
 * written directly from the paper's definitions.
 *
 * Paper: "Approximating Softmax in Pretrained LLMs: Model Sensitivity and
 * Kernel Acceleration".  Sections cited:
 *   App. A.1, Eq. (exact-attention)        softmax over the valid key set
 *   Sec. 5.2 Eq. (m-h15) = App. B.1 Eq. (h15)  the Rowmax-H15 weight
 *   App. B.1 "Implementation"              the FP32 add/shift realisation,
 *                                          clamp, doubled exponent constants,
 *                                          row sum and PV on the same weights
 *   App. B.1 "Relation to classical bit-level exponentiation"
 *                                          H = S o Q_1/2, octave-error envelope
 *   App. B.2 "Semantic simulation"         per-tile running max (tile 128),
 *                                          rescale threshold 0 (FP8 path)
 *   App. B.2, Table B2                     offline whole-row control
 *   App. A.6 Eq. (rowmax-pot)              Rowmax-PoT, K_max = 20
 *   App. B.2 "Exponential-map ablation"    the finer input-rounding family
 *                                          S(Q_{2^-k}(x)), k = 2, 3, realised
 *                                          with 2^k and a shift by 23 - k
 *
 * Precision policy: everything the paper leaves to "exact" arithmetic is done
 * in fp64 from the exactly decoded stored operands (bf16 values, or e4m3 codes
 * read as reals).  The steps that the paper fixes in FP32 (the exponent
 * argument, the add of 0x4B400000, the shift) are done in FP32 exactly as
 * stated.  Build with -ffp-contract=off and without -ffast-math.
 *
 * Parity status: every function here is pinned by tests against the paper's
 * worked example, closed forms, invariants, library routines or brute force,
 * except the items the paper leaves unpinned (H15 log-sum-exp, per-tile
 * element values, FP8 P rounding), which are pinned only by the definitions
 * written out below.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { OR_BF16 = 0, OR_FP8_E4M3 = 1 };
enum {
    OR_EXACT = 0,        /* App. A.1 exact softmax attention, fp64 */
    OR_H15_TILE = 1,     /* Rowmax-H15 with the per-tile running max (App. B.2) */
    OR_H15_WHOLEROW = 2, /* Rowmax-H15 anchored at the final whole-row max */
    OR_ROWMAX_POT = 3,   /* App. A.6 Rowmax-PoT, whole row, K_max = 20 */
    OR_EXACT_TILE = 4,   /* diagnostic: exact exp2 inside the same tile loop,
                            with the kernel's P storage rounding */
    OR_SQ4_TILE = 5,     /* S(Q_{1/4}(x)) with the per-tile running max */
    OR_SQ8_TILE = 6      /* S(Q_{1/8}(x)) with the per-tile running max */
};

static uint32_t f2u(float f) { uint32_t u; memcpy(&u, &f, 4); return u; }
static float u2f(uint32_t u) { float f; memcpy(&f, &u, 4); return f; }

int oracle_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* ---- operand decoding ------------------------------------------------- */

/* bfloat16: the top 16 bits of an IEEE binary32 pattern. */
double oracle_bf16_value(uint16_t b) { return (double)u2f((uint32_t)b << 16); }

/* OCP E4M3 ("e4m3fn"): sign, 4 exponent bits with bias 7, 3 mantissa bits,
 * subnormals at exponent field 0, no infinities, S.1111.111 is NaN. */
double oracle_e4m3_value(uint8_t c)
{
    int s = c >> 7, e = (c >> 3) & 15, m = c & 7;
    double v;
    if (e == 15 && m == 7) return NAN;
    if (e == 0) v = ldexp((double)m / 8.0, -6);
    else v = ldexp(1.0 + (double)m / 8.0, e - 7);
    return s ? -v : v;
}

/* Round to the nearest finite E4M3 value, ties to the code with an even
 * mantissa, saturating at +-448.  Brute force over every finite code. */
uint8_t oracle_e4m3_rne_satfinite(double x)
{
    if (isnan(x)) return 0x7F;
    uint8_t sign = signbit(x) ? 0x80 : 0x00;
    double a = fabs(x);
    if (a >= 448.0) return sign | 0x7E;
    int best = 0;
    double bestd = INFINITY;
    for (int c = 0; c <= 0x7E; c++) {
        double dd = fabs(oracle_e4m3_value((uint8_t)c) - a);
        if (dd < bestd || (dd == bestd && (c & 1) == 0)) { best = c; bestd = dd; }
    }
    return sign | (uint8_t)best;
}

/* Round an fp32 value to bfloat16 (round to nearest, ties to even). */
static uint16_t bf16_rne(float f)
{
    uint32_t u = f2u(f);
    uint32_t lsb = (u >> 16) & 1u;
    return (uint16_t)((u + 0x7FFFu + lsb) >> 16);
}

/* ---- the Rowmax-H15 weight -------------------------------------------- */

/* App. B.1 "Implementation".  y is the doubled base-two exponent 2x in FP32.
 * Clamp at -252 (so the exponent field cannot wrap), add 0x4B400000 =
 * 2^23 + 2^22 with an FP32 round-to-nearest-even add (this leaves
 * n = RNE(y) in the low mantissa bits), shift left by 22 (bit 0 of n becomes
 * the leading mantissa bit, the rest lands in the exponent field) and add the
 * bit pattern of 1.0, all modulo 2^32. */
float oracle_h15_weight(float y)
{
    volatile float yc = (y < -252.0f) ? -252.0f : y;
    volatile float t = yc + 12582912.0f; /* 0x4B400000 as a float */
    uint32_t u = (f2u(t) << 22) + 0x3F800000u;
    return u2f(u);
}

/* Sec. 5.2 Eq. (m-h15) written out with library rounding: n = RNE(2x),
 * weight = (1 + (n mod 2)/2) * 2^floor(n/2), floor toward -inf and the
 * non-negative residue.  The argument is y = 2x. */
double oracle_h15_ideal(double y)
{
    double n = nearbyint(y); /* default rounding mode: nearest, ties to even */
    double k = floor(n / 2.0);
    double r = n - 2.0 * k;
    return (1.0 + 0.5 * r) * ldexp(1.0, (int)k);
}

/* Exhaustive comparison of the two forms above over every fp32 y in
 * [lo, hi], both taken after the clamp at -252.  Returns the number of
 * mismatching bit patterns; *count receives the number of values tested. */
int64_t oracle_h15_exhaustive(float lo, float hi, int64_t* count)
{
    int64_t bad = 0, n = 0;
    /* positive half: patterns 0x00000000 .. bits(hi); negative half:
     * 0x80000000 .. bits(lo).  Walk both ranges of integer patterns. */
    uint32_t hi_bits = hi >= 0 ? f2u(hi) : 0;
    uint32_t lo_mag = lo <= 0 ? (f2u(lo) & 0x7FFFFFFFu) : 0;
    int64_t npos = hi >= 0 ? (int64_t)hi_bits + 1 : 0;
    int64_t nneg = lo <= 0 ? (int64_t)lo_mag + 1 : 0;
    int64_t total = npos + nneg;
#pragma omp parallel for reduction(+ : bad, n) schedule(static)
    for (int64_t idx = 0; idx < total; idx++) {
        uint32_t bits = idx < npos ? (uint32_t)idx : (0x80000000u | (uint32_t)(idx - npos));
        float y = u2f(bits);
        if (y < lo || y > hi) continue;
        double yc = y < -252.0f ? -252.0 : (double)y;
        float want = (float)oracle_h15_ideal(yc);
        float got = oracle_h15_weight(y);
        n++;
        if (f2u(want) != f2u(got)) bad++;
    }
    if (count) *count = n;
    return bad;
}

/* ---- the S(Q_{2^-k}) family (App. B.2 "Exponential-map ablation") ------ */

/* The realisation that the paper's bit-level test describes: the FP32 add of
 * 0x4B400000 and shift of App. B.1, with the input scaled by 2^k instead of
 * 2 and the result shifted left by 23 - k.  y is 2^k x in FP32; the clamp x >= -126 becomes
 * y >= -126 * 2^k.  k = 1 is Rowmax-H15.  Valid for 0 <= k <= 22 and
 * |y| < 2^22. */
float oracle_sq_weight(float y, int k)
{
    const float lo = -126.0f * (float)(1 << k);
    volatile float yc = (y < lo) ? lo : y;
    volatile float t = yc + 12582912.0f;
    uint32_t u = (f2u(t) << (23 - k)) + 0x3F800000u;
    return u2f(u);
}

/* The ideal operator written from its two definitions: the unshifted
 * Schraudolph map S(q) = 2^floor(q) (1 + q - floor(q)) (App. B.1, "Relation
 * to classical bit-level exponentiation") applied to the quantised input
 * Q_{2^-k}(x) = 2^-k RNE(2^k x).  The argument is y = 2^k x. */
double oracle_sq_ideal(double y, int k)
{
    double q = ldexp(nearbyint(y), -k); /* RNE in the default rounding mode */
    double fl = floor(q);
    return ldexp(1.0 + (q - fl), (int)fl);
}

/* Exhaustive comparison of the two forms above over every fp32 y in
 * [lo, hi], both taken after the clamp at -126 * 2^k.  Returns the number of
 * mismatching bit patterns; *count receives the number of values tested. */
int64_t oracle_sq_exhaustive(float lo, float hi, int k, int64_t* count)
{
    int64_t bad = 0, n = 0;
    const double clamp = -126.0 * (double)(1 << k);
    uint32_t hi_bits = hi >= 0 ? f2u(hi) : 0;
    uint32_t lo_mag = lo <= 0 ? (f2u(lo) & 0x7FFFFFFFu) : 0;
    int64_t npos = hi >= 0 ? (int64_t)hi_bits + 1 : 0;
    int64_t nneg = lo <= 0 ? (int64_t)lo_mag + 1 : 0;
    int64_t total = npos + nneg;
#pragma omp parallel for reduction(+ : bad, n) schedule(static)
    for (int64_t idx = 0; idx < total; idx++) {
        uint32_t bits = idx < npos ? (uint32_t)idx : (0x80000000u | (uint32_t)(idx - npos));
        float y = u2f(bits);
        if (y < lo || y > hi) continue;
        double yc = (double)y < clamp ? clamp : (double)y;
        float want = (float)oracle_sq_ideal(yc, k);
        float got = oracle_sq_weight(y, k);
        n++;
        if (f2u(want) != f2u(got)) bad++;
    }
    if (count) *count = n;
    return bad;
}

/* The same comparison on a given list of base-two exponents x (fp32): both
 * forms are evaluated at y = 2^k x after the clamp x >= -126 (the scaling by
 * 2^k is exact).  Returns the number of mismatching bit patterns. */
int64_t oracle_sq_count_mismatch(const float* x, int64_t n, int k)
{
    int64_t bad = 0;
#pragma omp parallel for reduction(+ : bad) schedule(static)
    for (int64_t i = 0; i < n; i++) {
        float xc = x[i] < -126.0f ? -126.0f : x[i];
        float y = ldexpf(xc, k);
        float want = (float)oracle_sq_ideal((double)y, k);
        float got = oracle_sq_weight(y, k);
        if (f2u(want) != f2u(got)) bad++;
    }
    return bad;
}

/* The exponent-path constant: the base-two scale applied to a raw logit,
 * c1 = fp32(scale * q_descale * k_descale * log2(e)), products taken in
 * double in this order.  The H15 path uses c2 = 2*c1 (App. B.1: separate,
 * doubled exponent-path constants). */
float oracle_c1(double scale, double qd, double kd)
{
    return (float)(scale * qd * kd * 1.4426950408889634);
}

/* ---- one row of the tiled online-softmax recurrence -------------------- */

/* Rowmax-H15 (or the exact-exp2 diagnostic) for one query row, following
 * App. B.1 / B.2: keys are visited in tiles of Bc in increasing order; for
 * each tile the running max m is moved to m_new (threshold tau in base-two
 * units; tau = 0 always moves it to max(m, tile max)); the running sum and
 * the output accumulator are rescaled by alpha = 2^((m - m_new) c1); the
 * weight of each valid key is computed from the doubled exponent
 * y = fma(s, c2, fma(-m_new, c2, 2 off)), and the row sum and PV consume the
 * same weights (P is W stored in the operand type).  Masked keys carry
 * W = P = 0 and never enter the max.
 *   s      fp32 raw logits of the row, length S
 *   vrows  decoded V rows [S][d] (NULL: no O accumulation)
 *   jend   number of valid keys (keys 0 .. jend-1), >= 1
 * Outputs (each optional): o[d] (unscaled by vd), *lse, w[S], p[S]. */
/* The anchor rule of App. B.2 "Conditional rescaling moves the anchor": the
 * running max moves to max(m, mt) only when it grows by more than tau in
 * base-two units, (mt - m) c1 > tau, evaluated in FP32 like the rest of the
 * exponent path; with tau = 0 this is always max(m, mt).  The first tile with
 * a valid key always sets the anchor. */
static int grows(float mt, float m, float c1, double tau)
{
    if (m == -INFINITY) return 1;
    volatile float dm = mt - m;
    volatile float g = dm * c1;
    return g > (float)tau;
}

/* One pass of the per-tile recurrence over the keys [j0, j1) of a row, its
 * tiles [j0 + t Bc, j0 + (t+1) Bc) taken in increasing order; keys at or
 * beyond jend are masked (W = P = 0, never in the max) and the pass stops at
 * the first tile that starts at or beyond jend.  The running max starts at
 * -inf.  On return *m_out is the pass's final anchor (-inf when it saw no
 * valid key), *l_out its running sum and acc[d] its output accumulator, both
 * relative to that anchor (acc unscaled by vd).
 *   s      fp32 raw logits of the row, indexed by key
 *   vrows  decoded V rows, indexed by key ([key][d]; NULL: no accumulation)
 *   move   optional per-tile decisions (1: move the anchor to max(m, mt)),
 *          indexed by the pass's tile number, used for a decision shared by a
 *          group of rows; NULL: this row's own test with tau.
 * Optional per-key outputs (written for the pass's valid keys only): w, p,
 * y (the fp32 exponent argument the weight is taken from, before any clamp)
 * and anchor (the running max the key's tile used). */
static void tile_pass(const float* s, const double* vrows, int d, int j0, int j1, int jend, float c1,
                      int off, int Bc, double tau, const uint8_t* move, int dtype, int exact_exp, int kq,
                      float* m_out, double* l_out, double* acc, float* w, uint32_t* p, float* y, float* anchor)
{
    /* the input-rounding exponent k: 1 for Rowmax-H15 (c2 = 2 c1, shift 22),
     * 2 or 3 for S(Q_{2^-k}) (2^k c1, shift 23 - k); the scaling by 2^k is exact */
    const float ck = ldexpf(c1, kq);
    float m = -INFINITY;
    double l = 0.0;
    if (acc) for (int c = 0; c < d; c++) acc[c] = 0.0;
    for (int t0 = j0; t0 < j1 && t0 < jend; t0 += Bc) {
        int t1 = t0 + Bc < j1 ? t0 + Bc : j1;
        int v1 = t1 < jend ? t1 : jend;
        float mt = -INFINITY;
        for (int j = t0; j < v1; j++) mt = fmaxf(mt, s[j]);
        int mv = move ? (m == -INFINITY || move[(t0 - j0) / Bc]) : grows(mt, m, c1, tau);
        float m_new = mv ? fmaxf(m, mt) : m;
        double alpha = (m == -INFINITY) ? 0.0 : exp2(((double)m - (double)m_new) * (double)c1);
        l *= alpha;
        if (acc) for (int c = 0; c < d; c++) acc[c] *= alpha;
        float nbk = fmaf(-m_new, ck, (float)((1 << kq) * off));
        float nb1 = fmaf(-m_new, c1, (float)off);
        for (int j = t0; j < v1; j++) {
            float wj, yj;
            if (exact_exp) {
                yj = fmaf(s[j], c1, nb1);
                wj = (float)exp2((double)yj);
            } else {
                yj = fmaf(s[j], ck, nbk);
                wj = kq == 1 ? oracle_h15_weight(yj) : oracle_sq_weight(yj, kq);
            }
            uint32_t pb;
            double pv;
            if (dtype == OR_BF16) {
                pb = bf16_rne(wj);
                pv = oracle_bf16_value((uint16_t)pb);
            } else {
                pb = oracle_e4m3_rne_satfinite((double)wj);
                pv = oracle_e4m3_value((uint8_t)pb);
            }
            l += (double)wj;
            if (acc && vrows)
                for (int c = 0; c < d; c++) acc[c] += pv * vrows[(size_t)j * d + c];
            if (w) w[j] = wj;
            if (p) p[j] = pb;
            if (y) y[j] = yj;
            if (anchor) anchor[j] = m_new;
        }
        m = m_new;
    }
    *m_out = m;
    *l_out = l;
}

/* The whole row as one pass (keys 0 .. S-1, valid below jend >= 1), then
 * O = acc / l * vd and LSE = ln2 (m c1 + log2 l - off).  Per-key outputs of
 * masked keys are W = P = 0, y = anchor = -inf. */
static void tiled_row(const float* s, const double* vrows, int S, int d, int jend, float c1,
                      int off, int Bc, double tau, const uint8_t* move, int dtype, int exact_exp,
                      int kq, double vd, double* o, double* lse, float* w, uint32_t* p, double* acc,
                      float* y, float* anchor)
{
    for (int j = 0; j < S; j++) {
        if (w) w[j] = 0.0f;
        if (p) p[j] = 0u;
        if (y) y[j] = -INFINITY;
        if (anchor) anchor[j] = -INFINITY;
    }
    float m;
    double l;
    tile_pass(s, vrows, d, 0, S, jend, c1, off, Bc, tau, move, dtype, exact_exp, kq, &m, &l, acc, w, p, y,
              anchor);
    if (o && acc)
        for (int c = 0; c < d; c++) o[c] = acc[c] / l * vd;
    if (lse) *lse = M_LN2 * ((double)m * (double)c1 + log2(l) - (double)off);
}

/* W and P of one row from given fp32 logits (for bit-exact comparison with
 * values that another implementation stored for the same logits). */
int oracle_sq_row_from_logits(const float* s, int S, int i, int causal, float c1, int dtype,
                              int Bc, double tau, int exact_exp, int k, float* w_out,
                              uint32_t* p_out, double* lse_out)
{
    if (S <= 0 || Bc <= 0 || i < 0 || i >= S || k < 1 || k > 3) return -1;
    int off = dtype == OR_FP8_E4M3 ? 8 : 0;
    int jend = causal ? i + 1 : S;
    tiled_row(s, NULL, S, 0, jend, c1, off, Bc, tau, NULL, dtype, exact_exp, k, 1.0, NULL, lse_out, w_out,
              p_out, NULL, NULL, NULL);
    return 0;
}

/* As oracle_sq_row_from_logits with the per-tile anchor decisions given
 * (move[t] for tile t), for rows that share a group decision. */
int oracle_sq_row_from_logits_moves(const float* s, int S, int i, int causal, float c1, int dtype,
                                    int Bc, const uint8_t* move, int k, float* w_out,
                                    uint32_t* p_out, double* lse_out)
{
    if (S <= 0 || Bc <= 0 || i < 0 || i >= S || k < 1 || k > 3 || !move) return -1;
    int off = dtype == OR_FP8_E4M3 ? 8 : 0;
    int jend = causal ? i + 1 : S;
    tiled_row(s, NULL, S, 0, jend, c1, off, Bc, 0.0, move, dtype, 0, k, 1.0, NULL, lse_out, w_out,
              p_out, NULL, NULL, NULL);
    return 0;
}

/* The per-key exponent arguments of one row from given fp32 logits: y[j] is
 * the fp32 value the weight of key j is taken from (2^k x for the lattice
 * weights, x for the exact exponential; before the clamp) and anchor[j] the
 * running max of its tile; masked keys get -inf in both.  w[j] as in
 * oracle_sq_row_from_logits.  (A test uses them to bound how far a weight
 * can move when the logits move: a lattice weight changes only where y
 * crosses a rounding boundary.) */
int oracle_sq_row_exponents_from_logits(const float* s, int S, int i, int causal, float c1, int dtype,
                                        int Bc, int exact_exp, int k, float* y_out, float* anchor_out,
                                        float* w_out)
{
    if (S <= 0 || Bc <= 0 || i < 0 || i >= S || k < 1 || k > 3 || !y_out || !anchor_out) return -1;
    int off = dtype == OR_FP8_E4M3 ? 8 : 0;
    int jend = causal ? i + 1 : S;
    tiled_row(s, NULL, S, 0, jend, c1, off, Bc, 0.0, NULL, dtype, exact_exp, k, 1.0, NULL, NULL, w_out,
              NULL, NULL, y_out, anchor_out);
    return 0;
}

/* Rowmax-PoT (App. A.6 Eq. (rowmax-pot)) of one query row from its fp32
 * logits, in the arithmetic a kernel can reproduce: the anchor m is the
 * row's maximum raw logit over its valid keys, the base-two gap is
 * x_j = fp32(fp32(m - s_j) * c1) (the paper's Delta_j / ln 2 with
 * c1 = fp32(scale qd kd log2 e)), d_j = min(K_max, floor(x_j + 1/2)) with
 * K_max = 20 (x_j + 1/2 is exact in fp32 below 2^22), w_j = 2^-d_j, and
 * masked keys carry w = P = 0.  P is w in the operand type (BF16 only: every
 * level 2^0 .. 2^-20 is exact there).  l sums w; LSE = ln2 (m c1 + log2 l). */
int oracle_pot_row_from_logits(const float* s, int S, int i, int causal, float c1, float* w_out,
                               uint32_t* p_out, double* lse_out)
{
    if (S <= 0 || i < 0 || i >= S) return -1;
    const int jend = causal ? i + 1 : S;
    float m = -INFINITY;
    for (int j = 0; j < jend; j++) m = fmaxf(m, s[j]);
    double l = 0.0;
    for (int j = 0; j < S; j++) {
        float w = 0.0f;
        if (j < jend) {
            volatile float gap = m - s[j];
            volatile float x = gap * c1;
            volatile float t = x + 0.5f;
            float d = floorf(t);
            if (d > 20.0f) d = 20.0f;
            w = ldexpf(1.0f, -(int)d);
        }
        l += (double)w;
        if (w_out) w_out[j] = w;
        if (p_out) p_out[j] = bf16_rne(w);
    }
    if (lse_out) *lse_out = M_LN2 * ((double)m * (double)c1 + log2(l));
    return 0;
}

int oracle_h15_row_from_logits(const float* s, int S, int i, int causal, float c1, int dtype,
                               int Bc, double tau, int exact_exp, float* w_out, uint32_t* p_out,
                               double* lse_out)
{
    return oracle_sq_row_from_logits(s, S, i, causal, c1, dtype, Bc, tau, exact_exp, 1, w_out,
                                     p_out, lse_out);
}

/* ---- the anchor decision shared by a group of rows ---------------------- */

static double decode(const void* base, size_t idx, int dtype);

/* FlashAttention-4 takes the conditional-rescale decision per warp of 32
 * query rows (App. B.2, "Semantic simulation": the simulation decides per
 * row, the kernel per warp of 32 rows): every row of the group moves its
 * anchor to max(m, mt) when any row's anchor grows by more than tau.  The
 * per-tile decisions (move[t] for tile t) of rows [i0, i1) from their fp32
 * logits (row r of the group at s + r * S). */
int oracle_group_moves_from_logits(const float* s, int S, int i0, int i1, int causal, float c1,
                                   int Bc, double tau, uint8_t* move)
{
    if (S <= 0 || Bc <= 0 || i0 < 0 || i1 <= i0 || i1 > S || !move) return -1;
    const int n = i1 - i0;
    float* m = malloc(sizeof(float) * (size_t)n);
    float* mt = malloc(sizeof(float) * (size_t)n);
    if (!m || !mt) {
        free(m); free(mt);
        return -3;
    }
    for (int r = 0; r < n; r++) m[r] = -INFINITY;
    for (int t = 0; t * Bc < S; t++) {
        int any = 0;
        for (int r = 0; r < n; r++) {
            const int jend = causal ? i0 + r + 1 : S;
            const int t0 = t * Bc, t1 = (t0 + Bc < jend) ? t0 + Bc : jend;
            mt[r] = -INFINITY;
            for (int j = t0; j < t1; j++) mt[r] = fmaxf(mt[r], s[(size_t)r * S + j]);
            if (mt[r] != -INFINITY && grows(mt[r], m[r], c1, tau)) any = 1;
        }
        move[t] = (uint8_t)any;
        for (int r = 0; r < n; r++)
            if (m[r] == -INFINITY || any) m[r] = fmaxf(m[r], mt[r]);
    }
    free(m); free(mt);
    return 0;
}

/* The same decisions for rows [i0, i1) of head (b, h) of stored operands. */
static int group_moves(const void* q, const void* k, int dtype, int Hq, int Hkv, int S, int d,
                       int b, int h, int i0, int i1, int causal, float c1, int Bc, double tau,
                       uint8_t* move)
{
    const int n = i1 - i0, hk = h / (Hq / Hkv);
    const size_t kvoff = ((size_t)b * Hkv + hk) * S * d;
    float* s32 = malloc(sizeof(float) * (size_t)n * S);
    double* qrow = malloc(sizeof(double) * d);
    if (!s32 || !qrow) {
        free(s32); free(qrow);
        return -3;
    }
    for (int r = 0; r < n; r++) {
        const size_t qoff = (((size_t)b * Hq + h) * S + i0 + r) * d;
        for (int c = 0; c < d; c++) qrow[c] = decode(q, qoff + c, dtype);
        for (int j = 0; j < S; j++) {
            double dot = 0.0;
            for (int c = 0; c < d; c++) dot += qrow[c] * decode(k, kvoff + (size_t)j * d + c, dtype);
            s32[(size_t)r * S + j] = (float)dot;
        }
    }
    const int rc = oracle_group_moves_from_logits(s32, S, i0, i1, causal, c1, Bc, tau, move);
    free(s32); free(qrow);
    return rc;
}

/* ---- full attention --------------------------------------------------- */

static double decode(const void* base, size_t idx, int dtype)
{
    if (dtype == OR_BF16) return oracle_bf16_value(((const uint16_t*)base)[idx]);
    return oracle_e4m3_value(((const uint8_t*)base)[idx]);
}

/* Attention forward for the listed rows (flat index (b*Hq + h)*S + i), or
 * for all B*Hq*S rows when rows == NULL.  q: [B][Hq][S][d]; k, v:
 * [B][Hkv][S][d], stored as bf16 bit patterns (uint16) or e4m3 codes
 * (uint8).  Query head h reads key/value head h / (Hq/Hkv).  Causal means
 * query i sees keys j <= i.  o receives nrows x d doubles, lse nrows
 * doubles (natural log of the normaliser of the scaled logits).
 * Returns 0, -1 on invalid arguments, or -3 when memory ran out. */
int oracle_attn(const void* q, const void* k, const void* v, int dtype, double qd, double kd,
                double vd, int B, int Hq, int Hkv, int S, int d, int causal, double scale, int mode,
                int Bc, double tau, int tau_group, const int64_t* rows, int64_t nrows, double* o,
                double* lse)
{
    if (tau_group < 1) return -1;
    if (!q || !k || !v || !o || B <= 0 || Hq <= 0 || Hkv <= 0 || S <= 0 || d <= 0) return -1;
    if (Hq % Hkv != 0 || (dtype != OR_BF16 && dtype != OR_FP8_E4M3) || mode < 0 || mode > 6)
        return -1;
    if (mode != OR_EXACT && mode != OR_ROWMAX_POT && mode != OR_H15_WHOLEROW && Bc <= 0) return -1;
    const int64_t total = (int64_t)B * Hq * S;
    if (!rows) nrows = total;
    const int group = Hq / Hkv;
    const double sigma = scale * qd * kd; /* natural-log scale of a raw logit */
    const float c1 = oracle_c1(scale, qd, kd);
    const int off = dtype == OR_FP8_E4M3 ? 8 : 0;
    int bad = 0, nomem = 0;
#pragma omp parallel for schedule(dynamic, 4) reduction(| : bad, nomem)
    for (int64_t r = 0; r < nrows; r++) {
        int64_t flat = rows ? rows[r] : r;
        if (flat < 0 || flat >= total) { bad = 1; continue; }
        const int i = (int)(flat % S);
        const int h = (int)((flat / S) % Hq);
        const int b = (int)(flat / ((int64_t)S * Hq));
        const int hk = h / group;
        const size_t qoff = (((size_t)b * Hq + h) * S + i) * d;
        const size_t kvoff = ((size_t)b * Hkv + hk) * S * d;
        const int jend = causal ? i + 1 : S;

        double* qrow = malloc(sizeof(double) * d);
        double* sexact = malloc(sizeof(double) * S);
        double* vrows = malloc(sizeof(double) * (size_t)jend * d);
        double* acc = malloc(sizeof(double) * d);
        float* s32 = malloc(sizeof(float) * S);
        if (!qrow || !sexact || !vrows || !acc || !s32) {
            free(qrow); free(sexact); free(vrows); free(acc); free(s32);
            nomem = 1;
            continue;
        }
        for (int c = 0; c < d; c++) qrow[c] = decode(q, qoff + c, dtype);
        for (int j = 0; j < jend; j++) {
            double dot = 0.0;
            for (int c = 0; c < d; c++) dot += qrow[c] * decode(k, kvoff + (size_t)j * d + c, dtype);
            sexact[j] = dot;
            s32[j] = (float)dot; /* the raw logit, rounded once to fp32 */
            for (int c = 0; c < d; c++) vrows[(size_t)j * d + c] = decode(v, kvoff + (size_t)j * d + c, dtype);
        }
        for (int j = jend; j < S; j++) s32[j] = 0.0f; /* never read: masked */
        double* orow = o + (size_t)r * d;

        if (mode == OR_EXACT || mode == OR_ROWMAX_POT) {
            double smax = -INFINITY;
            for (int j = 0; j < jend; j++) smax = fmax(smax, sexact[j]);
            double den = 0.0;
            for (int c = 0; c < d; c++) acc[c] = 0.0;
            for (int j = 0; j < jend; j++) {
                double wj;
                if (mode == OR_EXACT) {
                    wj = exp(-sigma * (smax - sexact[j])); /* w_j = exp(-Delta_j) */
                } else {
                    double xj = sigma * (smax - sexact[j]) / M_LN2; /* x_j = Delta_j / ln 2 */
                    double dj = floor(xj + 0.5);
                    if (dj > 20.0) dj = 20.0; /* K_max = 20 */
                    wj = ldexp(1.0, -(int)dj);
                }
                den += wj;
                for (int c = 0; c < d; c++) acc[c] += wj * vrows[(size_t)j * d + c];
            }
            for (int c = 0; c < d; c++) orow[c] = acc[c] / den * vd;
            if (lse) lse[r] = sigma * smax + log(den);
        } else {
            int tile = (mode == OR_H15_WHOLEROW) ? S : Bc;
            int kq = mode == OR_SQ4_TILE ? 2 : mode == OR_SQ8_TILE ? 3 : 1;
            uint8_t* move = NULL;
            if (tau_group > 1) {
                const int i0 = i / tau_group * tau_group;
                const int i1 = i0 + tau_group < S ? i0 + tau_group : S;
                move = malloc((size_t)(S / tile + 1));
                if (!move || group_moves(q, k, dtype, Hq, Hkv, S, d, b, h, i0, i1, causal, c1, tile, tau,
                                         move) != 0) {
                    free(move); free(qrow); free(sexact); free(vrows); free(acc); free(s32);
                    nomem = 1;
                    continue;
                }
            }
            tiled_row(s32, vrows, S, d, jend, c1, off, tile, tau, move, dtype, mode == OR_EXACT_TILE, kq,
                      vd, orow, lse ? &lse[r] : NULL, NULL, NULL, acc, NULL, NULL);
            free(move);
        }
        free(qrow); free(sexact); free(vrows); free(acc); free(s32);
    }
    return bad ? -1 : nomem ? -3 : 0;
}

/* Raw fp32 logits s_ij = fp32(sum_c q_ic k_jc) of one query row (exact fp64
 * sum of the decoded operands, rounded once).  Keys j > i are still written
 * (the caller decides about masking). */
int oracle_logits_row(const void* q, const void* k, int dtype, int B, int Hq, int Hkv, int S, int d,
                      int b, int h, int i, float* s_out)
{
    if (!q || !k || !s_out || b < 0 || b >= B || h < 0 || h >= Hq || i < 0 || i >= S) return -1;
    if (Hkv <= 0 || Hq % Hkv) return -1;
    const int hk = h / (Hq / Hkv);
    const size_t qoff = (((size_t)b * Hq + h) * S + i) * d;
    const size_t kvoff = ((size_t)b * Hkv + hk) * S * d;
    for (int j = 0; j < S; j++) {
        double dot = 0.0;
        for (int c = 0; c < d; c++)
            dot += decode(q, qoff + c, dtype) * decode(k, kvoff + (size_t)j * d + c, dtype);
        s_out[j] = (float)dot;
    }
    return 0;
}

/* ---- decode over a key/value cache ------------------------------------ */

/* The paper states attention for square inputs (App. A.1: one query row per
 * key position) and leaves decode out of its scope; this is the extension
 * the library implements.  Sq query rows per head attend to the first Sk
 * rows of a key/value cache; query position i sees keys j <= Sk - Sq + i
 * when causal (bottom-right alignment: the last query row sees the whole
 * cache, and with Sq = Sk this is the square causal mask), every key
 * otherwise.
 *
 * The keys are cut into consecutive parts of split_keys keys (a positive
 * multiple of Bc; 0 or >= Sk: one part).  Within each part the per-tile
 * recurrence of App. B.1 / B.2 runs on its own: its tiles start at the
 * part's first key and its running max starts at -inf, so the weights of a
 * part are taken relative to the part's own running maxima.  The parts then
 * merge exactly (the softmax identity, fp64):
 *     m = max_p m_p,   f_p = 2^(c1 (m_p - m)),
 *     l = sum_p f_p l_p,   acc = sum_p f_p acc_p,
 *     O = acc / l * vd,    LSE = ln2 (m c1 + log2 l - off),
 * parts without a visible key taking no part.  With one part this is the
 * whole row's recurrence (tiled_row).  EXACT mode is the plain softmax over
 * the visible keys, which no cut changes. */
static void decode_row(const float* s32, const double* vrows, int Sk, int d, int jend, float c1, int off,
                       int Bc, int split_keys, int dtype, int exact_exp, int kq, double vd, double* o,
                       double* lse, float* w, uint32_t* p, double* acc, double* part_acc)
{
    const int part = (split_keys <= 0 || split_keys >= Sk) ? Sk : split_keys;
    for (int j = 0; j < Sk; j++) {
        if (w) w[j] = 0.0f;
        if (p) p[j] = 0u;
    }
    /* the merged maximum first, then every part rescaled to it */
    const int nparts = (Sk + part - 1) / part;
    float m = -INFINITY;
    for (int j = 0; j < jend; j++) m = fmaxf(m, s32[j]);
    double l = 0.0;
    if (acc) for (int c = 0; c < d; c++) acc[c] = 0.0;
    for (int pi = 0; pi < nparts; pi++) {
        const int j0 = pi * part, j1 = j0 + part < Sk ? j0 + part : Sk;
        if (j0 >= jend) break; /* no visible key in this part or any later one */
        float mp;
        double lp;
        tile_pass(s32, vrows, d, j0, j1, jend, c1, off, Bc, 0.0, NULL, dtype, exact_exp, kq, &mp, &lp,
                  part_acc, w, p, NULL, NULL);
        const double f = exp2(((double)mp - (double)m) * (double)c1);
        l += f * lp;
        if (acc && part_acc)
            for (int c = 0; c < d; c++) acc[c] += f * part_acc[c];
    }
    if (o && acc)
        for (int c = 0; c < d; c++) o[c] = acc[c] / l * vd;
    if (lse) *lse = M_LN2 * ((double)m * (double)c1 + log2(l) - (double)off);
}

/* Decode attention for the listed rows (flat index (b*Hq + h)*Sq + i), or for
 * all B*Hq*Sq rows when rows == NULL.  q: [B][Hq][Sq][d]; k, v:
 * [B][Hkv][Sk_cap][d] of which the first Sk rows of every head are the cache
 * (bf16 bit patterns or e4m3 codes).  Modes: OR_EXACT, OR_H15_TILE,
 * OR_SQ4_TILE, OR_SQ8_TILE, OR_EXACT_TILE.  o receives nrows x d doubles, lse
 * nrows doubles.  Returns 0, -1 on invalid arguments (including
 * Sq > Sk, Sk > Sk_cap, or a split_keys that is not a multiple of Bc), or -3
 * when memory ran out. */
int oracle_decode(const void* q, const void* k, const void* v, int dtype, double qd, double kd, double vd,
                  int B, int Hq, int Hkv, int Sq, int Sk, int Sk_cap, int d, int causal, double scale,
                  int mode, int Bc, int split_keys, const int64_t* rows, int64_t nrows, double* o,
                  double* lse)
{
    if (!q || !k || !v || !o || B <= 0 || Hq <= 0 || Hkv <= 0 || Sq <= 0 || Sk <= 0 || d <= 0) return -1;
    if (Hq % Hkv != 0 || Sq > Sk || Sk > Sk_cap || Bc <= 0 || split_keys < 0 || split_keys % Bc != 0)
        return -1;
    if (dtype != OR_BF16 && dtype != OR_FP8_E4M3) return -1;
    if (mode != OR_EXACT && mode != OR_H15_TILE && mode != OR_SQ4_TILE && mode != OR_SQ8_TILE &&
        mode != OR_EXACT_TILE)
        return -1;
    const int64_t total = (int64_t)B * Hq * Sq;
    if (!rows) nrows = total;
    const int group = Hq / Hkv;
    const double sigma = scale * qd * kd;
    const float c1 = oracle_c1(scale, qd, kd);
    const int off = dtype == OR_FP8_E4M3 ? 8 : 0;
    const int kq = mode == OR_SQ4_TILE ? 2 : mode == OR_SQ8_TILE ? 3 : 1;
    int bad = 0, nomem = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : bad, nomem)
    for (int64_t r = 0; r < nrows; r++) {
        int64_t flat = rows ? rows[r] : r;
        if (flat < 0 || flat >= total) { bad = 1; continue; }
        const int i = (int)(flat % Sq);
        const int h = (int)((flat / Sq) % Hq);
        const int b = (int)(flat / ((int64_t)Sq * Hq));
        const int hk = h / group;
        const size_t qoff = (((size_t)b * Hq + h) * Sq + i) * d;
        const size_t kvoff = ((size_t)b * Hkv + hk) * (size_t)Sk_cap * d;
        const int jend = causal ? Sk - Sq + i + 1 : Sk;
        double* qrow = malloc(sizeof(double) * d);
        double* sexact = malloc(sizeof(double) * Sk);
        double* vrows = malloc(sizeof(double) * (size_t)jend * d);
        double* acc = malloc(sizeof(double) * d);
        double* part_acc = malloc(sizeof(double) * d);
        float* s32 = malloc(sizeof(float) * Sk);
        if (!qrow || !sexact || !vrows || !acc || !part_acc || !s32) {
            free(qrow); free(sexact); free(vrows); free(acc); free(part_acc); free(s32);
            nomem = 1;
            continue;
        }
        for (int c = 0; c < d; c++) qrow[c] = decode(q, qoff + c, dtype);
        for (int j = 0; j < jend; j++) {
            double dot = 0.0;
            for (int c = 0; c < d; c++) dot += qrow[c] * decode(k, kvoff + (size_t)j * d + c, dtype);
            sexact[j] = dot;
            s32[j] = (float)dot;
            for (int c = 0; c < d; c++) vrows[(size_t)j * d + c] = decode(v, kvoff + (size_t)j * d + c, dtype);
        }
        for (int j = jend; j < Sk; j++) s32[j] = 0.0f; /* never read: masked */
        double* orow = o + (size_t)r * d;
        if (mode == OR_EXACT) {
            double smax = -INFINITY;
            for (int j = 0; j < jend; j++) smax = fmax(smax, sexact[j]);
            double den = 0.0;
            for (int c = 0; c < d; c++) acc[c] = 0.0;
            for (int j = 0; j < jend; j++) {
                const double wj = exp(-sigma * (smax - sexact[j]));
                den += wj;
                for (int c = 0; c < d; c++) acc[c] += wj * vrows[(size_t)j * d + c];
            }
            for (int c = 0; c < d; c++) orow[c] = acc[c] / den * vd;
            if (lse) lse[r] = sigma * smax + log(den);
        } else {
            decode_row(s32, vrows, Sk, d, jend, c1, off, Bc, split_keys, dtype, mode == OR_EXACT_TILE, kq, vd,
                       orow, lse ? &lse[r] : NULL, NULL, NULL, acc, part_acc);
        }
        free(qrow); free(sexact); free(vrows); free(acc); free(part_acc); free(s32);
    }
    return bad ? -1 : nomem ? -3 : 0;
}

/* W and P of one decode row from given fp32 logits s[0 .. Sk-1] with the
 * part semantics of oracle_decode (jend visible keys), and its LSE. */
int oracle_decode_row_from_logits(const float* s, int Sk, int jend, float c1, int dtype, int Bc,
                                  int split_keys, int exact_exp, int k, float* w_out, uint32_t* p_out,
                                  double* lse_out)
{
    if (Sk <= 0 || jend < 1 || jend > Sk || Bc <= 0 || split_keys < 0 || split_keys % Bc != 0 || k < 1 ||
        k > 3)
        return -1;
    const int off = dtype == OR_FP8_E4M3 ? 8 : 0;
    decode_row(s, NULL, Sk, 0, jend, c1, off, Bc, split_keys, dtype, exact_exp, k, 1.0, NULL, lse_out, w_out,
               p_out, NULL, NULL);
    return 0;
}

/* Raw fp32 logits of one decode row (exact fp64 dot products of the stored
 * operands, rounded once), layouts as in oracle_decode. */
int oracle_decode_logits_row(const void* q, const void* k, int dtype, int B, int Hq, int Hkv, int Sq, int Sk,
                             int Sk_cap, int d, int b, int h, int i, float* s_out)
{
    if (!q || !k || !s_out || b < 0 || b >= B || h < 0 || h >= Hq || i < 0 || i >= Sq || Hkv <= 0 ||
        Hq % Hkv || Sk > Sk_cap)
        return -1;
    const int hk = h / (Hq / Hkv);
    const size_t qoff = (((size_t)b * Hq + h) * Sq + i) * d;
    const size_t kvoff = ((size_t)b * Hkv + hk) * (size_t)Sk_cap * d;
    for (int j = 0; j < Sk; j++) {
        double dot = 0.0;
        for (int c = 0; c < d; c++)
            dot += decode(q, qoff + c, dtype) * decode(k, kvoff + (size_t)j * d + c, dtype);
        s_out[j] = (float)dot;
    }
    return 0;
}
