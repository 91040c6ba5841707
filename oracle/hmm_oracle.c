/*
 * hmm_oracle.c -- plain scalar CPU oracle for Plan7 profile-HMM database
 * search: MSV (uint8) filter -> Viterbi (int16) filter with int32 rescore
 * -> Forward (fp64 here).
 *
 * TEST INFRASTRUCTURE.  Only the test suite, the package smoke check and the
 * benchmark's CPU-baseline leg may load this library.  It shares no code,
 * header, table or constant generator with the GPU library; both are written
 * independently from the same model definition.
 *
 * What is computed.  The paper (ParaFold, Background section) names the
 * jackhmmer searches of UniRef90 and MGnify as the CPU-bound core of the
 * MSA-construction stage; the core of such a search is scoring one Plan7
 * profile HMM against every database sequence.  The paper does not print
 * the recurrences, score systems or filter thresholds, so this file fixes
 * them explicitly ("readings", each stated where it is used):
 *
 *  Model (nats).  Alphabet of 20 residues, codes 0..19.  Match scores
 *  msc_k(a) = ln(e_k(a)/f(a)) for k = 1..M, insert scores
 *  isc_k(a) = ln(i_k(a)/f(a)) for k = 1..M-1.  Node transitions
 *  MM MI MD IM II DM DD out of nodes 1..M-1 (natural logs; -inf if 0).
 *  Local multihit configuration for target length L:
 *    B->M_k entry ln(2/(M(M+1))) for every k; M_k->E and D_k->E score 0;
 *    E->C = E->J = ln 1/2; N->N = J->J = C->C = ln(L/(L+3));
 *    N->B = J->B = C->T = ln(3/(L+3)).  N, C, J emit with score 0.
 *
 *  Float recurrences (Viterbi: max, Forward: log-sum-exp), row i, a = x_i:
 *    M_k(i) = msc_k(a) + OP{ M_{k-1}(i-1)+MM_{k-1}, I_{k-1}(i-1)+IM_{k-1},
 *                            D_{k-1}(i-1)+DM_{k-1}, B(i-1)+ENTRY }
 *    I_k(i) = isc_k(a) + OP{ M_k(i-1)+MI_k, I_k(i-1)+II_k }
 *    D_k(i) = OP{ M_{k-1}(i)+MD_{k-1}, D_{k-1}(i)+DD_{k-1} }     (D_1 = -inf)
 *    E(i) = OP_k{ M_k(i), D_k(i) }
 *    J(i) = OP{ J(i-1)+LOOP, E(i)+EJ }, C(i) = OP{ C(i-1)+LOOP, E(i)+EC }
 *    N(i) = N(i-1)+LOOP, B(i) = OP{ N(i)+MOVE, J(i)+MOVE }
 *    with N(0) = 0, B(0) = MOVE, everything else -inf; score = C(L)+MOVE.
 *
 *  Integer filters: see orc_msv and orc_vit16 / orc_vit32 below.
 *
 * Build: gcc -O2 -fno-tree-vectorize -shared -fPIC (scalar on purpose).
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <time.h>

#define KA 20                       /* alphabet size */
#define ORC_S8 (3.0 / M_LN2)        /* MSV units per nat: third-bits */
#define ORC_S16 (500.0 / M_LN2)     /* Viterbi units per nat: 1/500 bits */
#define ORC_BASE8 190               /* MSV offset for the N/J start */
#define ORC_NEG16 (-32768)
#define ORC_NEG32 (-1073741824)     /* -2^30: int32 "minus infinity" floor */

/* flag bits, per target */
#define F_MSV_PASS 0x01
#define F_MSV_OVF 0x02
#define F_VIT_RAN 0x04
#define F_VIT_PASS 0x08
#define F_VIT_OVF 0x10
#define F_FWD_RAN 0x20
#define F_FWD_PASS 0x40
#define F_BIAS_PASS 0x80             /* passed the composition-bias filter (only when it is on) */

/* Composition-bias null model: switch probability between its two states */
#define ORC_BIAS_SWITCH (1.0 / 64.0)

typedef struct orc_profile {
  int M;
  double entry;                     /* ln(2/(M(M+1))) */
  double *msc;                      /* [M][KA]   node k at row k-1 */
  double *isc;                      /* [M-1][KA] */
  double *tr;                       /* [M-1][7]  MM MI MD IM II DM DD */
  /* MSV tables */
  int bias8, entry8, exit8;
  uint8_t *cost8;                   /* [M][KA] */
  /* Viterbi tables */
  int entry16, ej16;
  int16_t *msc16, *isc16, *t16;     /* [M][KA], [M-1][KA], [M-1][7] */
  /* composition-bias filter: ln of (mean match emission / background) */
  double bias_lr[KA];
} orc_profile;

/* Rounding used for every quantised score: q(x) = floor(x + 1/2), fp64. */
static long qround(double x) { return (long)floor(x + 0.5); }
static long clampl(long v, long lo, long hi) { return v < lo ? lo : (v > hi ? hi : v); }

void orc_profile_free(orc_profile *p) {
  if (!p) return;
  free(p->msc); free(p->isc); free(p->tr);
  free(p->cost8); free(p->msc16); free(p->isc16); free(p->t16);
  free(p);
}

/*
 * Build scores and integer tables from probabilities.
 *   match[M][20], insert[M-1][20], trans[M-1][7], bg[20]; row-major fp64.
 * MSV (uint8, third-bits): sc8 = q(S8*ln(e/f)); BIAS8 = clamp(-min sc8, 0,
 *   255); COST8 = clamp(BIAS8 - sc8, 0, 255); ENTRY8 = q(-S8*ENTRY);
 *   EXIT8 = q(S8*ln 2).
 * Viterbi (int16, 1/500 bits): msc16/isc16 = sat16(q(S16*score));
 *   t16 = sat16(q(S16*ln t)), or -32768 when t = 0; ENTRY16 = q(S16*ENTRY);
 *   EJ16 = q(S16*ln 1/2).
 */
orc_profile *orc_profile_new(int M, const double *bg, const double *match,
                             const double *insert, const double *trans) {
  if (M < 1) return NULL;
  orc_profile *p = calloc(1, sizeof *p);
  if (!p) return NULL;
  int Mi = M - 1;
  p->M = M;
  p->msc = malloc(sizeof(double) * M * KA);
  p->isc = malloc(sizeof(double) * (Mi > 0 ? Mi : 1) * KA);
  p->tr = malloc(sizeof(double) * (Mi > 0 ? Mi : 1) * 7);
  p->cost8 = malloc((size_t)M * KA);
  p->msc16 = malloc(sizeof(int16_t) * M * KA);
  p->isc16 = malloc(sizeof(int16_t) * (Mi > 0 ? Mi : 1) * KA);
  p->t16 = malloc(sizeof(int16_t) * (Mi > 0 ? Mi : 1) * 7);
  if (!p->msc || !p->isc || !p->tr || !p->cost8 || !p->msc16 || !p->isc16 || !p->t16) {
    orc_profile_free(p);
    return NULL;
  }
  p->entry = log(2.0 / ((double)M * ((double)M + 1.0)));
  for (int k = 0; k < M; k++)
    for (int a = 0; a < KA; a++) p->msc[k * KA + a] = log(match[k * KA + a] / bg[a]);
  for (int k = 0; k < Mi; k++)
    for (int a = 0; a < KA; a++) p->isc[k * KA + a] = log(insert[k * KA + a] / bg[a]);
  for (int k = 0; k < Mi; k++)
    for (int t = 0; t < 7; t++) p->tr[k * 7 + t] = log(trans[k * 7 + t]);

  /* MSV */
  long minsc = 0;
  long *sc8 = malloc(sizeof(long) * M * KA);
  if (!sc8) { orc_profile_free(p); return NULL; }
  for (int i = 0; i < M * KA; i++) {
    sc8[i] = qround(ORC_S8 * p->msc[i]);
    if (i == 0 || sc8[i] < minsc) minsc = sc8[i];
  }
  p->bias8 = (int)clampl(-minsc, 0, 255);
  for (int i = 0; i < M * KA; i++) p->cost8[i] = (uint8_t)clampl(p->bias8 - sc8[i], 0, 255);
  free(sc8);
  p->entry8 = (int)clampl(qround(-ORC_S8 * p->entry), 0, 255);
  p->exit8 = (int)clampl(qround(ORC_S8 * log(2.0)), 0, 255);

  /* Viterbi */
  for (int i = 0; i < M * KA; i++)
    p->msc16[i] = (int16_t)clampl(qround(ORC_S16 * p->msc[i]), -32768, 32767);
  /* a zero insert probability scores -inf: the int16 floor */
  for (int i = 0; i < Mi * KA; i++)
    p->isc16[i] = insert[i] > 0.0 ? (int16_t)clampl(qround(ORC_S16 * p->isc[i]), -32768, 32767)
                                  : (int16_t)ORC_NEG16;
  for (int i = 0; i < Mi * 7; i++)
    p->t16[i] = trans[i] > 0.0 ? (int16_t)clampl(qround(ORC_S16 * p->tr[i]), -32768, 32767)
                               : (int16_t)ORC_NEG16;
  p->entry16 = (int)clampl(qround(ORC_S16 * p->entry), -32768, 32767);
  p->ej16 = (int)clampl(qround(ORC_S16 * log(0.5)), -32768, 32767);
  /* mean match composition over the nodes, as odds against the background */
  for (int a = 0; a < KA; a++) {
    double m = 0.0;
    for (int k = 0; k < M; k++) m += match[k * KA + a];
    p->bias_lr[a] = log(m / (double)M / bg[a]);
  }
  return p;
}

int orc_profile_M(const orc_profile *p) { return p->M; }

/* scalars: bias8, entry8, exit8, entry16, ej16 */
void orc_profile_scalars(const orc_profile *p, int32_t *out) {
  out[0] = p->bias8; out[1] = p->entry8; out[2] = p->exit8;
  out[3] = p->entry16; out[4] = p->ej16;
}

void orc_profile_tables(const orc_profile *p, uint8_t *cost8, int16_t *msc16,
                        int16_t *isc16, int16_t *t16) {
  int M = p->M, Mi = M - 1;
  if (cost8) memcpy(cost8, p->cost8, (size_t)M * KA);
  if (msc16) memcpy(msc16, p->msc16, sizeof(int16_t) * M * KA);
  if (isc16 && Mi > 0) memcpy(isc16, p->isc16, sizeof(int16_t) * Mi * KA);
  if (t16 && Mi > 0) memcpy(t16, p->t16, sizeof(int16_t) * Mi * 7);
}

/* Length-model parameters for target length L (>= 1):
 *   LOOP = ln(L/(L+3)), MOVE = ln(3/(L+3)); MOVE8 = clamp(q(-S8*MOVE), 0,
 *   255); MOVE16 = sat16(q(S16*MOVE)); NULL(L) = L ln(L/(L+1)) + ln(1/(L+1))
 *   is the null model's log-likelihood offset (nats, residue terms excluded). */
double orc_loop(int L) { return log((double)L / ((double)L + 3.0)); }
double orc_move(int L) { return log(3.0 / ((double)L + 3.0)); }
int orc_move8(int L) { return (int)clampl(qround(-ORC_S8 * orc_move(L)), 0, 255); }
int orc_move16(int L) { return (int)clampl(qround(ORC_S16 * orc_move(L)), -32768, 32767); }
double orc_null(int L) {
  return (double)L * log((double)L / ((double)L + 1.0)) + log(1.0 / ((double)L + 1.0));
}

/*
 * Score cutoffs from P-value thresholds (readings: lambda = ln 2 per bit;
 * MSV and Viterbi bit scores follow a Gumbel law P(S > x) = 1 -
 * exp(-exp(-lambda (x - mu))); Forward bit scores an exponential tail
 * P(S > x) = exp(-lambda (x - tau)); a target passes when P < F, and F >= 1
 * passes everything).
 *   msv bits = ((raw - BASE8)/S8 - 3 - NULL(L)) / ln 2
 *   vit bits = (vit/S16 - 3 - NULL(L)) / ln 2
 *   fwd bits = (fwd_nats - NULL(L)) / ln 2
 * The constant 3 nats stands for the N/C/J loop scores that the integer
 * filters omit.  The integer cutoffs are the smallest integers whose bit
 * score exceeds the cutoff, so the pass test is an exact integer compare.
 *   calib = {mu_msv, mu_vit, tau} (bits), F = {F1, F2, F3}
 *   out: thr8 (0..256), thr16 (int32), fwd_thr (nats; pass if fwd > it)
 */
void orc_thresholds(const double *calib, const double *F, int L, int32_t *thr8,
                    int32_t *thr16, double *fwd_thr) {
  double nul = orc_null(L);
  if (F[0] >= 1.0) {
    *thr8 = 0;
  } else {
    double x1 = calib[0] - log(-log(1.0 - F[0])) / M_LN2;
    double y = floor(ORC_BASE8 + ORC_S8 * (x1 * M_LN2 + nul + 3.0)) + 1.0;
    *thr8 = (int32_t)(y < 0.0 ? 0.0 : (y > 256.0 ? 256.0 : y));
  }
  if (F[1] >= 1.0) {
    *thr16 = INT32_MIN;
  } else {
    double x2 = calib[1] - log(-log(1.0 - F[1])) / M_LN2;
    double y = floor(ORC_S16 * (x2 * M_LN2 + nul + 3.0)) + 1.0;
    *thr16 = (int32_t)(y < -2147483647.0 ? -2147483647.0 : (y > 2147483647.0 ? 2147483647.0 : y));
  }
  if (F[2] >= 1.0)
    *fwd_thr = -INFINITY;
  else
    *fwd_thr = (calib[2] - log(F[2]) / M_LN2) * M_LN2 + nul;
}

/* ---------------------------------------------------------------- MSV */

static int sadd8(int a, int b) { int r = a + b; return r > 255 ? 255 : r; }
static int ssub8(int a, int b) { int r = a - b; return r < 0 ? 0 : r; }

/*
 * MSV filter: multi-segment ungapped local alignment in saturating uint8
 * arithmetic ("+" saturates at 255, "-" at 0).  Per row i, a = x_i, with
 * mm[0] = 0 and previous-row values on the right:
 *    xBe   = xB - ENTRY8
 *    mm[k] = (max(mm[k-1], xBe) + BIAS8) - COST8_k(a)      k = 1..M
 *    xE    = max_k mm[k];   overflow if xE >= 255 - BIAS8
 *    xJ    = max(xJ, xE - EXIT8)
 *    xB    = max(BASE8 - MOVE8, xJ - MOVE8)
 * starting from mm = 0, xJ = 0, xB = BASE8 - MOVE8.  The N, C and J loop
 * scores are omitted (0), and C equals J because E->C = E->J.
 * Returns msv_raw = 255 on overflow, else xJ - MOVE8.
 */
int orc_msv(const orc_profile *p, const uint8_t *x, int L, int *ovf_out) {
  int M = p->M;
  int *mm = calloc((size_t)M + 1, sizeof(int));
  int mv = orc_move8(L);
  int base = ssub8(ORC_BASE8, mv);
  int xJ = 0, xB = base, ovf = 0;
  for (int i = 0; i < L; i++) {
    const uint8_t a = x[i];
    int xBe = ssub8(xB, p->entry8);
    int xE = 0;
    for (int k = M; k >= 1; k--) {   /* descending: mm[k-1] is still the previous row */
      int v = mm[k - 1] > xBe ? mm[k - 1] : xBe;
      mm[k] = ssub8(sadd8(v, p->bias8), p->cost8[(k - 1) * KA + a]);
      if (mm[k] > xE) xE = mm[k];
    }
    if (xE >= 255 - p->bias8) { ovf = 1; break; }
    int e = ssub8(xE, p->exit8);
    if (e > xJ) xJ = e;
    int jb = ssub8(xJ, mv);
    xB = jb > base ? jb : base;
  }
  free(mm);
  if (ovf_out) *ovf_out = ovf;
  return ovf ? 255 : ssub8(xJ, mv);
}

/* ---------------------------------------------------------------- Viterbi */

static int sat16(int v) { return v < -32768 ? -32768 : (v > 32767 ? 32767 : v); }
static int fl32(long v) { return v < ORC_NEG32 ? ORC_NEG32 : (int)v; }

static int imax(int a, int b) { return a > b ? a : b; }

/*
 * Viterbi filter, int16 saturating (1/500-bit units), and its int32 rescore.
 * Every add saturates on its own (sat16), max is exact.  Per row, with
 * previous-row Mp, Ip, Dp, xBp:
 *    M_k = sat(max(sat(xBp+ENTRY16), sat(Mp_{k-1}+MM_{k-1}),
 *                  sat(Ip_{k-1}+IM_{k-1}), sat(Dp_{k-1}+DM_{k-1})) + msc_k(a))
 *          (k = 1: the B term only)
 *    I_k = sat(max(sat(Mp_k+MI_k), sat(Ip_k+II_k)) + isc_k(a))     k < M
 *    D_1 = -inf; D_k = max(sat(M_{k-1}+MD_{k-1}), sat(D_{k-1}+DD_{k-1}))
 *    overflow if some M_k or I_k equals 32767
 *    xE = max_k max(M_k, D_k); xJ = max(xJ, sat(xE+EJ16))
 *    xB = max(sat(MOVE16), sat(xJ+MOVE16))
 * from M = I = D = xJ = -32768 and xB = sat(MOVE16).  Loops score 0.
 * Result: 32767 on overflow, else sat(xJ + MOVE16).
 *
 * The int32 rescore is the same recurrence in int32 with every add floored
 * at -2^30 (no upper clamp): result xJ + MOVE16.
 */
static long vit_generic(const orc_profile *p, const uint8_t *x, int L, int wide, int *ovf_out) {
  int M = p->M;
  int neg = wide ? ORC_NEG32 : ORC_NEG16;
  int *Mp = malloc(sizeof(int) * (M + 1)), *Ip = malloc(sizeof(int) * (M + 1));
  int *Dp = malloc(sizeof(int) * (M + 1)), *Mc = malloc(sizeof(int) * (M + 1));
  int *Ic = malloc(sizeof(int) * (M + 1)), *Dc = malloc(sizeof(int) * (M + 1));
  for (int k = 0; k <= M; k++) Mp[k] = Ip[k] = Dp[k] = neg;
  int mv = orc_move16(L);
#define ADD(a, b) (wide ? fl32((long)(a) + (long)(b)) : sat16((a) + (b)))
  int xJ = neg;
  int xB = ADD(0, mv);
  int ovf = 0;
  for (int i = 0; i < L; i++) {
    const int a = x[i];
    int xBe = ADD(xB, p->entry16);
    for (int k = 1; k <= M; k++) {
      int m = xBe;
      if (k > 1) {
        const int16_t *t = p->t16 + (k - 2) * 7;      /* node k-1 */
        m = imax(m, ADD(Mp[k - 1], t[0]));
        m = imax(m, ADD(Ip[k - 1], t[3]));
        m = imax(m, ADD(Dp[k - 1], t[5]));
      }
      Mc[k] = ADD(m, p->msc16[(k - 1) * KA + a]);
      if (k < M) {
        const int16_t *t = p->t16 + (k - 1) * 7;      /* node k */
        int v = imax(ADD(Mp[k], t[1]), ADD(Ip[k], t[4]));
        Ic[k] = ADD(v, p->isc16[(k - 1) * KA + a]);
      } else {
        Ic[k] = neg;
      }
    }
    Dc[1] = neg;
    for (int k = 2; k <= M; k++) {
      const int16_t *t = p->t16 + (k - 2) * 7;        /* node k-1 */
      Dc[k] = imax(ADD(Mc[k - 1], t[2]), ADD(Dc[k - 1], t[6]));
    }
    int xE = neg;
    for (int k = 1; k <= M; k++) {
      if (!wide && (Mc[k] == 32767 || (k < M && Ic[k] == 32767))) ovf = 1;
      xE = imax(xE, imax(Mc[k], Dc[k]));
    }
    xJ = imax(xJ, ADD(xE, p->ej16));
    xB = imax(ADD(0, mv), ADD(xJ, mv));
    int *tmp;
    tmp = Mp; Mp = Mc; Mc = tmp;
    tmp = Ip; Ip = Ic; Ic = tmp;
    tmp = Dp; Dp = Dc; Dc = tmp;
  }
  long res = ADD(xJ, mv);
#undef ADD
  free(Mp); free(Ip); free(Dp); free(Mc); free(Ic); free(Dc);
  if (ovf_out) *ovf_out = ovf;
  if (!wide && ovf) return 32767;
  return res;
}

int orc_vit16(const orc_profile *p, const uint8_t *x, int L, int *ovf) {
  return (int)vit_generic(p, x, L, 0, ovf);
}

int32_t orc_vit32(const orc_profile *p, const uint8_t *x, int L) {
  return (int32_t)vit_generic(p, x, L, 1, NULL);
}

/* ---------------------------------------------------------------- float DP */

static double lse(double a, double b) {
  if (a == -INFINITY) return b;
  if (b == -INFINITY) return a;
  double m = a > b ? a : b;
  return m + log1p(exp(-fabs(a - b)));
}
static double dmax(double a, double b) { return a > b ? a : b; }

/* The float recurrences of the header comment, in log space; use_max
 * selects Viterbi (max over paths) or Forward (log-sum over paths). */
static double float_dp(const orc_profile *p, const uint8_t *x, int L, int use_max) {
  int M = p->M;
  double (*op)(double, double) = use_max ? dmax : lse;
  double loop = orc_loop(L), move = orc_move(L), half = log(0.5);
  double *Mp = malloc(sizeof(double) * (M + 1)), *Ip = malloc(sizeof(double) * (M + 1));
  double *Dp = malloc(sizeof(double) * (M + 1)), *Mc = malloc(sizeof(double) * (M + 1));
  double *Ic = malloc(sizeof(double) * (M + 1)), *Dc = malloc(sizeof(double) * (M + 1));
  for (int k = 0; k <= M; k++) Mp[k] = Ip[k] = Dp[k] = -INFINITY;
  double N = 0.0, B = move, J = -INFINITY, C = -INFINITY;
  for (int i = 0; i < L; i++) {
    const int a = x[i];
    for (int k = 1; k <= M; k++) {
      double m = B + p->entry;
      if (k > 1) {
        const double *t = p->tr + (k - 2) * 7;
        m = op(m, Mp[k - 1] + t[0]);
        m = op(m, Ip[k - 1] + t[3]);
        m = op(m, Dp[k - 1] + t[5]);
      }
      Mc[k] = m + p->msc[(k - 1) * KA + a];
      if (k < M) {
        const double *t = p->tr + (k - 1) * 7;
        Ic[k] = p->isc[(k - 1) * KA + a] + op(Mp[k] + t[1], Ip[k] + t[4]);
      } else {
        Ic[k] = -INFINITY;
      }
    }
    Dc[1] = -INFINITY;
    for (int k = 2; k <= M; k++) {
      const double *t = p->tr + (k - 2) * 7;
      Dc[k] = op(Mc[k - 1] + t[2], Dc[k - 1] + t[6]);
    }
    double E = -INFINITY;
    for (int k = 1; k <= M; k++) E = op(op(E, Mc[k]), Dc[k]);
    J = op(J + loop, E + half);
    C = op(C + loop, E + half);
    N = N + loop;
    B = op(N + move, J + move);
    double *tmp;
    tmp = Mp; Mp = Mc; Mc = tmp;
    tmp = Ip; Ip = Ic; Ic = tmp;
    tmp = Dp; Dp = Dc; Dc = tmp;
  }
  free(Mp); free(Ip); free(Dp); free(Mc); free(Ic); free(Dc);
  return C + move;
}

double orc_vit_f64(const orc_profile *p, const uint8_t *x, int L) { return float_dp(p, x, L, 1); }
double orc_fwd_f64(const orc_profile *p, const uint8_t *x, int L) { return float_dp(p, x, L, 0); }

/*
 * Second, independent Forward formulation: probability space in fp64 with
 * an exact power-of-two rescale after every row (the exponent of the largest
 * special-state value), the removed exponents summed as an integer.
 * Result ln(C(L) * exp(MOVE)) + (sum of exponents) * ln 2.
 */
double orc_fwd_f64_scaled(const orc_profile *p, const uint8_t *x, int L) {
  int M = p->M;
  double loop = (double)L / ((double)L + 3.0), move = 3.0 / ((double)L + 3.0);
  double entry = 2.0 / ((double)M * ((double)M + 1.0));
  double *em = malloc(sizeof(double) * M * KA), *ei = malloc(sizeof(double) * (M > 1 ? M - 1 : 1) * KA);
  double *tp = malloc(sizeof(double) * (M > 1 ? M - 1 : 1) * 7);
  for (int i = 0; i < M * KA; i++) em[i] = exp(p->msc[i]);
  for (int i = 0; i < (M - 1) * KA; i++) ei[i] = exp(p->isc[i]);
  for (int i = 0; i < (M - 1) * 7; i++) tp[i] = exp(p->tr[i]);
  double *Mp = calloc(M + 1, sizeof(double)), *Ip = calloc(M + 1, sizeof(double));
  double *Dp = calloc(M + 1, sizeof(double)), *Mc = calloc(M + 1, sizeof(double));
  double *Ic = calloc(M + 1, sizeof(double)), *Dc = calloc(M + 1, sizeof(double));
  double N = 1.0, B = move, J = 0.0, C = 0.0;
  long shift = 0;
  for (int i = 0; i < L; i++) {
    const int a = x[i];
    for (int k = 1; k <= M; k++) {
      double m = B * entry;
      if (k > 1) {
        const double *t = tp + (k - 2) * 7;
        m += Mp[k - 1] * t[0] + Ip[k - 1] * t[3] + Dp[k - 1] * t[5];
      }
      Mc[k] = m * em[(k - 1) * KA + a];
      if (k < M) {
        const double *t = tp + (k - 1) * 7;
        Ic[k] = (Mp[k] * t[1] + Ip[k] * t[4]) * ei[(k - 1) * KA + a];
      } else {
        Ic[k] = 0.0;
      }
    }
    Dc[1] = 0.0;
    for (int k = 2; k <= M; k++) {
      const double *t = tp + (k - 2) * 7;
      Dc[k] = Mc[k - 1] * t[2] + Dc[k - 1] * t[6];
    }
    double E = 0.0;
    for (int k = 1; k <= M; k++) E += Mc[k] + Dc[k];
    J = J * loop + E * 0.5;
    C = C * loop + E * 0.5;
    N = N * loop;
    B = (N + J) * move;
    double big = E;
    if (J > big) big = J;
    if (C > big) big = C;
    if (N > big) big = N;
    if (B > big) big = B;
    if (big > 0.0) {
      int ex;
      frexp(big, &ex);
      double s = ldexp(1.0, -ex);
      for (int k = 1; k <= M; k++) { Mc[k] *= s; Ic[k] *= s; Dc[k] *= s; }
      J *= s; C *= s; N *= s; B *= s;
      shift += ex;
    }
    double *tmp;
    tmp = Mp; Mp = Mc; Mc = tmp;
    tmp = Ip; Ip = Ic; Ic = tmp;
    tmp = Dp; Dp = Dc; Dc = tmp;
  }
  double res = log(C * move) + (double)shift * M_LN2;
  free(em); free(ei); free(tp);
  free(Mp); free(Ip); free(Dp); free(Mc); free(Ic); free(Dc);
  return res;
}

/* ---------------------------------------------------------------- composition bias
 *
 * Composition-bias filter (reading): a null model with two states, R
 * emitting the background f and S emitting the profile's mean match
 * composition m(a) = (1/M) sum_k e_k(a); it starts in R or S with
 * probability 1 - w, w and switches state with probability w at every
 * further residue (w = 1/64).  The bias score is its log-likelihood ratio
 * against the background (nats):
 *    beta(x) = ln sum over state paths of P(path) prod_i r_{s_i}(x_i),
 *    r_R = 1, r_S(a) = m(a)/f(a).
 * With the filter on, a target that passes MSV goes on to Viterbi only if
 * MSV overflowed or  msv_raw - S8 * max(beta, 0) >= THR8(L)  (the MSV
 * score, less the bias in MSV units, still reaches the MSV cutoff).
 * Forward recursion in log space over the two states.
 */
double orc_bias(const orc_profile *p, const uint8_t *x, int L) {
  const double ls = log(ORC_BIAS_SWITCH), lt = log1p(-ORC_BIAS_SWITCH);
  double aR = lt, aS = ls + p->bias_lr[x[0]];
  for (int i = 1; i < L; i++) {
    const double r = lse(aR + lt, aS + ls);
    const double q = lse(aR + ls, aS + lt) + p->bias_lr[x[i]];
    aR = r;
    aS = q;
  }
  return lse(aR, aS);
}

/* ---------------------------------------------------------------- search */

typedef struct {
  const orc_profile *p;
  const uint8_t *res;
  const int64_t *off;
  int64_t n;
  const int32_t *thr8, *thr16;
  const double *fthr;
  int all_f3;
  int fwd_scaled;
  int bias;
  double *beta;
  int16_t *msv;
  int32_t *vit;
  double *fwd;
  uint8_t *flags;
  int64_t next;                     /* work counter (atomic) */
  double stage_s[3];
  pthread_mutex_t mu;
} search_job;

static double now_s(void) {
  struct timespec ts;
  clock_gettime(CLOCK_MONOTONIC, &ts);
  return ts.tv_sec + 1e-9 * ts.tv_nsec;
}

static void *search_worker(void *arg) {
  search_job *j = arg;
  double st[3] = {0, 0, 0};
  const int64_t chunk = 16;
  for (;;) {
    int64_t s = __atomic_fetch_add(&j->next, chunk, __ATOMIC_RELAXED);
    if (s >= j->n) break;
    int64_t e = s + chunk < j->n ? s + chunk : j->n;
    for (int64_t t = s; t < e; t++) {
      const uint8_t *x = j->res + j->off[t];
      int L = (int)(j->off[t + 1] - j->off[t]);
      double t0 = now_s();
      int ovf8 = 0;
      int raw = orc_msv(j->p, x, L, &ovf8);
      uint8_t fl = 0;
      if (ovf8) fl |= F_MSV_OVF;
      if (ovf8 || raw >= j->thr8[L]) fl |= F_MSV_PASS;
      j->msv[t] = (int16_t)raw;
      j->vit[t] = INT32_MIN;
      j->fwd[t] = NAN;
      int go = (fl & F_MSV_PASS) != 0;
      if (go && j->bias) {
        double b = orc_bias(j->p, x, L);
        if (j->beta) j->beta[t] = b;
        if (ovf8 || (double)raw - ORC_S8 * (b > 0.0 ? b : 0.0) >= (double)j->thr8[L]) fl |= F_BIAS_PASS;
        else go = 0;
      }
      double t1 = now_s();
      st[0] += t1 - t0;
      if (go) {
        int ovf16 = 0;
        int32_t v = orc_vit16(j->p, x, L, &ovf16);
        fl |= F_VIT_RAN;
        if (ovf16) {
          fl |= F_VIT_OVF;
          v = orc_vit32(j->p, x, L);
        }
        if (ovf16 || v >= j->thr16[L]) fl |= F_VIT_PASS;
        j->vit[t] = v;
        double t2 = now_s();
        st[1] += t2 - t1;
        if (fl & F_VIT_PASS) {
          double f = j->fwd_scaled ? orc_fwd_f64_scaled(j->p, x, L) : orc_fwd_f64(j->p, x, L);
          fl |= F_FWD_RAN;
          if (j->all_f3 || f > j->fthr[L]) fl |= F_FWD_PASS;
          j->fwd[t] = f;
          st[2] += now_s() - t2;
        }
      }
      j->flags[t] = fl;
    }
  }
  pthread_mutex_lock(&j->mu);
  for (int i = 0; i < 3; i++) j->stage_s[i] += st[i];
  pthread_mutex_unlock(&j->mu);
  return NULL;
}

/*
 * The filter pipeline over a database (caller order, results per target):
 * MSV on every target; Viterbi (int16, int32 rescore on overflow) on MSV
 * survivors; Forward on Viterbi survivors.  Targets not reaching a stage get
 * vit = INT32_MIN, fwd = NaN.  Flags as F_* above.
 *   res/off: concatenated residues and offsets[n+1]; calib = {mu_msv,
 *   mu_vit, tau}; F = {F1, F2, F3}; nthreads >= 1; stage_s[3] receives the
 *   summed per-thread seconds of each stage.  fwd_scaled selects the
 *   probability-space Forward formulation.  Returns 0, or -1 on bad input.
 */
int orc_search_bias(const orc_profile *p, const uint8_t *res, const int64_t *off, int64_t n,
                    const double *calib, const double *F, int nthreads, int fwd_scaled, int bias,
                    int16_t *msv, int32_t *vit, double *fwd, uint8_t *flags, double *beta, double *stage_s) {
  if (!p || n < 0 || nthreads < 1) return -1;
  int maxL = 1;
  for (int64_t t = 0; t < n; t++) {
    int64_t L = off[t + 1] - off[t];
    if (L < 1 || L > 1000000) return -1;
    if (L > maxL) maxL = (int)L;
  }
  int32_t *thr8 = malloc(sizeof(int32_t) * (maxL + 1));
  int32_t *thr16 = malloc(sizeof(int32_t) * (maxL + 1));
  double *fthr = malloc(sizeof(double) * (maxL + 1));
  for (int L = 1; L <= maxL; L++) orc_thresholds(calib, F, L, &thr8[L], &thr16[L], &fthr[L]);
  search_job j;
  memset(&j, 0, sizeof j);
  j.p = p; j.res = res; j.off = off; j.n = n;
  j.thr8 = thr8; j.thr16 = thr16; j.fthr = fthr; j.all_f3 = F[2] >= 1.0;
  j.fwd_scaled = fwd_scaled;
  j.bias = bias;
  j.beta = beta;
  if (beta) for (int64_t t = 0; t < n; t++) beta[t] = NAN;
  j.msv = msv; j.vit = vit; j.fwd = fwd; j.flags = flags;
  pthread_mutex_init(&j.mu, NULL);
  pthread_t *th = malloc(sizeof(pthread_t) * nthreads);
  for (int i = 0; i < nthreads; i++) pthread_create(&th[i], NULL, search_worker, &j);
  for (int i = 0; i < nthreads; i++) pthread_join(th[i], NULL);
  pthread_mutex_destroy(&j.mu);
  if (stage_s) for (int i = 0; i < 3; i++) stage_s[i] = j.stage_s[i];
  free(th); free(thr8); free(thr16); free(fthr);
  return 0;
}

/* ---------------------------------------------------------------- posterior decoding
 *
 * The step after the filter cascade: for a target that passed it, the
 * posterior probability of every state at every residue, from Forward and
 * Backward in fp64 log space (readings, stated here):
 *
 *  Backward, row i = L..0 (a = x_{i+1}; values are log P(rest | state at i)):
 *    bC(L) = MOVE;  bJ(L) = bN(L) = bB(L) = -inf
 *    bB(i) = OP_k { ENTRY + msc_k(a) + bM_k(i+1) }                   (i < L)
 *    bJ(i) = OP{ LOOP + bJ(i+1), MOVE + bB(i) };  bN likewise;  bC(i) = LOOP + bC(i+1)
 *    bE(i) = OP{ EC + bC(i), EJ + bJ(i) }
 *    bD_k(i) = OP{ bE(i), DM_k + msc_{k+1}(a) + bM_{k+1}(i+1), DD_k + bD_{k+1}(i) }
 *    bM_k(i) = OP{ bE(i), MM_k + msc_{k+1}(a) + bM_{k+1}(i+1),
 *                  MI_k + isc_k(a) + bI_k(i+1), MD_k + bD_{k+1}(i) }
 *    bI_k(i) = OP{ IM_k + msc_{k+1}(a) + bM_{k+1}(i+1), II_k + isc_k(a) + bI_k(i+1) }
 *    (terms through node k+1 or I_k exist for k < M only; row L has no
 *    emitting successor).  bN(0) equals the Forward total.
 *
 *  Posteriors, Z = Forward total (residue i = 1..L):
 *    P(M_k emits x_i) = exp(fM_k(i) + bM_k(i) - Z), I_k likewise;
 *    core(i) = sum_k of both;
 *    P(N emits x_i) = exp(fN(i) + bN(i) - Z)  (N occupied at row i >= 1);
 *    P(J emits x_i) = exp(fJ(i-1) + LOOP + bJ(i) - Z), C likewise;
 *    core + N + J + C = 1 at every residue;
 *    begin(i) = P(B at row i) = exp(fB(i) + bB(i) - Z), i = 0..L-1 (a domain
 *      starts at residue i+1);
 *    end(i) = P(E at row i) = exp(fE(i) + bE(i) - Z), i = 1..L (a domain
 *      ends at residue i).  Sum of begins = sum of ends = expected number of
 *      domains.
 */
int orc_decode(const orc_profile *p, const uint8_t *x, int L, double *tot, double *pcore,
               double *pnjc, double *pbeg, double *pend, double *pM, double *pI) {
  int M = p->M;
  if (L < 1) return -1;
  const double loop = orc_loop(L), move = orc_move(L), half = log(0.5);
  const size_t W = (size_t)M + 2;
  double *fM = malloc(sizeof(double) * (L + 1) * W), *fI = malloc(sizeof(double) * (L + 1) * W);
  double *sp = malloc(sizeof(double) * (L + 1) * 5);      /* fN fB fE fJ fC per row */
  double *Dp = malloc(sizeof(double) * W), *Dc = malloc(sizeof(double) * W);
  double *bMn = malloc(sizeof(double) * W), *bIn = malloc(sizeof(double) * W);
  double *bMc = malloc(sizeof(double) * W), *bIc = malloc(sizeof(double) * W);
  double *bDc = malloc(sizeof(double) * W);
  if (!fM || !fI || !sp || !Dp || !Dc || !bMn || !bIn || !bMc || !bIc || !bDc) {
    free(fM); free(fI); free(sp); free(Dp); free(Dc); free(bMn); free(bIn); free(bMc); free(bIc); free(bDc);
    return -1;
  }
#define FN(i) sp[(i) * 5 + 0]
#define FB(i) sp[(i) * 5 + 1]
#define FE(i) sp[(i) * 5 + 2]
#define FJ(i) sp[(i) * 5 + 3]
#define FC(i) sp[(i) * 5 + 4]
  for (size_t k = 0; k < W; k++) fM[k] = fI[k] = Dp[k] = -INFINITY;
  FN(0) = 0.0; FB(0) = move; FE(0) = FJ(0) = FC(0) = -INFINITY;
  for (int i = 1; i <= L; i++) {
    const int a = x[i - 1];
    double *Mp = fM + (size_t)(i - 1) * W, *Ip = fI + (size_t)(i - 1) * W;
    double *Mc = fM + (size_t)i * W, *Ic = fI + (size_t)i * W;
    Mc[0] = Ic[0] = Mc[M + 1] = Ic[M + 1] = -INFINITY;
    for (int k = 1; k <= M; k++) {
      double m = FB(i - 1) + p->entry;
      if (k > 1) {
        const double *t = p->tr + (k - 2) * 7;
        m = lse(m, Mp[k - 1] + t[0]);
        m = lse(m, Ip[k - 1] + t[3]);
        m = lse(m, Dp[k - 1] + t[5]);
      }
      Mc[k] = m + p->msc[(k - 1) * KA + a];
      if (k < M) {
        const double *t = p->tr + (k - 1) * 7;
        Ic[k] = p->isc[(k - 1) * KA + a] + lse(Mp[k] + t[1], Ip[k] + t[4]);
      } else {
        Ic[k] = -INFINITY;
      }
    }
    Dc[1] = -INFINITY;
    for (int k = 2; k <= M; k++) {
      const double *t = p->tr + (k - 2) * 7;
      Dc[k] = lse(Mc[k - 1] + t[2], Dc[k - 1] + t[6]);
    }
    double E = -INFINITY;
    for (int k = 1; k <= M; k++) E = lse(lse(E, Mc[k]), Dc[k]);
    FE(i) = E;
    FJ(i) = lse(FJ(i - 1) + loop, E + half);
    FC(i) = lse(FC(i - 1) + loop, E + half);
    FN(i) = FN(i - 1) + loop;
    FB(i) = lse(FN(i) + move, FJ(i) + move);
    double *tmp = Dp; Dp = Dc; Dc = tmp;
  }
  const double Z = FC(L) + move;

  /* Backward.  Row L first (no emitting successor), then rows L-1 .. 0. */
  double bC = move, bJ = -INFINITY, bN = -INFINITY, bB = -INFINITY;
  double bE = lse(half + bC, half + bJ);
  for (size_t k = 0; k < W; k++) bMc[k] = bIc[k] = bDc[k] = -INFINITY;
  for (int k = M; k >= 1; k--) {
    double dnext = k < M ? p->tr[(k - 1) * 7 + 6] + bDc[k + 1] : -INFINITY;
    double mdnext = k < M ? p->tr[(k - 1) * 7 + 2] + bDc[k + 1] : -INFINITY;
    bDc[k] = lse(bE, dnext);
    bMc[k] = lse(bE, mdnext);
    bIc[k] = -INFINITY;
  }
  for (int i = L;; i--) {
    /* posteriors of row i from the forward values and the backward row i */
    if (i >= 1) {
      const double *Mf = fM + (size_t)i * W, *If = fI + (size_t)i * W;
      double core = 0.0;
      for (int k = 1; k <= M; k++) {
        double pm = exp(Mf[k] + bMc[k] - Z);
        double pi = k < M ? exp(If[k] + bIc[k] - Z) : 0.0;
        if (pM) pM[(size_t)(i - 1) * M + (k - 1)] = pm;
        if (pI) pI[(size_t)(i - 1) * M + (k - 1)] = pi;
        core += pm + pi;
      }
      if (pcore) pcore[i - 1] = core;
      if (pnjc) {
        pnjc[3 * (i - 1) + 0] = exp(FN(i) + bN - Z);
        pnjc[3 * (i - 1) + 1] = exp(FJ(i - 1) + loop + bJ - Z);
        pnjc[3 * (i - 1) + 2] = exp(FC(i - 1) + loop + bC - Z);
      }
      if (pend) pend[i - 1] = exp(FE(i) + bE - Z);
    }
    if (i < L && pbeg) pbeg[i] = exp(FB(i) + bB - Z);
    if (i == 0) break;
    /* backward row i-1 from row i; a = x_i (1-based), the residue row i emitted */
    const int a = x[i - 1];
    double *tmp;
    tmp = bMn; bMn = bMc; bMc = tmp;
    tmp = bIn; bIn = bIc; bIc = tmp;
    double nB = -INFINITY;
    for (int k = 1; k <= M; k++) nB = lse(nB, p->entry + p->msc[(k - 1) * KA + a] + bMn[k]);
    bB = nB;
    bJ = lse(loop + bJ, move + bB);
    bN = lse(loop + bN, move + bB);
    bC = loop + bC;
    bE = lse(half + bC, half + bJ);
    bDc[M + 1] = -INFINITY;
    for (int k = M; k >= 1; k--) {
      if (k < M) {
        const double *t = p->tr + (k - 1) * 7;
        const double mn = p->msc[k * KA + a] + bMn[k + 1];
        const double in = p->isc[(k - 1) * KA + a] + bIn[k];
        bDc[k] = lse(bE, lse(t[5] + mn, t[6] + bDc[k + 1]));
        bMc[k] = lse(lse(bE, t[0] + mn), lse(t[1] + in, t[2] + bDc[k + 1]));
        bIc[k] = lse(t[3] + mn, t[4] + in);
      } else {
        bDc[k] = bE;
        bMc[k] = bE;
        bIc[k] = -INFINITY;
      }
    }
  }
  if (tot) { tot[0] = Z; tot[1] = bN; }
#undef FN
#undef FB
#undef FE
#undef FJ
#undef FC
  free(fM); free(fI); free(sp); free(Dp); free(Dc); free(bMn); free(bIn); free(bMc); free(bIc); free(bDc);
  return 0;
}

/*
 * Domain regions (reading): maximal runs of residues whose core posterior
 * is at least rt2, kept when some residue of the run reaches rt1.  Regions
 * are written as 1-based inclusive residue ranges se[2r], se[2r+1] (at most
 * cap of them); the return value is the number found.
 */
int orc_regions(const double *pcore, int L, double rt1, double rt2, int32_t *se, int cap) {
  int n = 0;
  for (int i = 0; i < L;) {
    if (!(pcore[i] >= rt2)) { i++; continue; }
    int j = i, hit = 0;
    while (j < L && pcore[j] >= rt2) { if (pcore[j] >= rt1) hit = 1; j++; }
    if (hit) {
      if (n < cap) { se[2 * n] = i + 1; se[2 * n + 1] = j; }
      n++;
    }
    i = j;
  }
  return n;
}

/*
 * Optimal-accuracy alignment of one region [s, e] (1-based, inclusive):
 * among single core paths B -> M_k1 ... M_k2 -> E that emit a contiguous
 * residue range [a, b] inside the region (transitions of zero probability
 * not allowed; the path starts and ends in a match state), maximise
 *    sum_{i in [a,b]} P(state of i emits x_i) + sum_{i in region, outside [a,b]} (1 - core(i)),
 * i.e. every residue earns the posterior of what the alignment says about
 * it: aligned to M_k / I_k, or not aligned to the model.
 * DP over rows i = s..e (G(i) = sum_{j=s}^{i} (1 - core(j))):
 *    OM_k(i) = pM_k(i) + max{ G(i-1), OM_{k-1}(i-1) [MM], OI_{k-1}(i-1) [IM], OD_{k-1}(i-1) [DM] }
 *    OI_k(i) = pI_k(i) + max{ OM_k(i-1) [MI], OI_k(i-1) [II] }          (k < M)
 *    OD_k(i) = max{ OM_{k-1}(i) [MD], OD_{k-1}(i) [DD] }                 (k >= 2)
 *    score = max_{i,k} OM_k(i) + G(e) - G(i)
 * Ties: the first candidate in the orders written above wins, the end cell
 * is the first maximum in row-major order.  Output code[i-s] for residues of
 * the region: +k (M_k), -k (I_k), 0 (not aligned); abk = {a, b, k1, k2}.
 * pM, pI: [L][M] posteriors of orc_decode.  Returns the score (or -inf if
 * the region is empty or no alignment exists).
 */
double orc_oa_align(const orc_profile *p, int L, const double *pcore, const double *pM, const double *pI,
                    int s, int e, int16_t *code, int32_t *abk) {
  const int M = p->M;
  if (s < 1 || e > L || s > e) return -INFINITY;
  const int R = e - s + 1;
  const size_t W = (size_t)M + 1;
  double *OMp = malloc(sizeof(double) * W), *OIp = malloc(sizeof(double) * W), *ODp = malloc(sizeof(double) * W);
  double *OMc = malloc(sizeof(double) * W), *OIc = malloc(sizeof(double) * W), *ODc = malloc(sizeof(double) * W);
  uint8_t *tb = malloc((size_t)R * W * 3);    /* per cell: M, I, D predecessor */
  double *G = malloc(sizeof(double) * (R + 1));
  if (!OMp || !OIp || !ODp || !OMc || !OIc || !ODc || !tb || !G) {
    free(OMp); free(OIp); free(ODp); free(OMc); free(OIc); free(ODc); free(tb); free(G);
    return -INFINITY;
  }
  enum { FROM_B = 0, FROM_M = 1, FROM_I = 2, FROM_D = 3 };
  G[0] = 0.0;
  for (int r = 0; r < R; r++) G[r + 1] = G[r] + (1.0 - pcore[s - 1 + r]);
  for (size_t k = 0; k < W; k++) OMp[k] = OIp[k] = ODp[k] = -INFINITY;
  double best = -INFINITY;
  int bi = -1, bk = -1;
  for (int r = 0; r < R; r++) {
    const int i = s + r;
    const double *pm = pM + (size_t)(i - 1) * M, *pi = pI + (size_t)(i - 1) * M;
    uint8_t *t = tb + (size_t)r * W * 3;
    OMc[0] = OIc[0] = ODc[0] = -INFINITY;
    for (int k = 1; k <= M; k++) {
      double v = G[r];
      int from = FROM_B;
      if (k > 1 && r > 0) {
        const double *tr = p->tr + (k - 2) * 7;
        if (tr[0] > -INFINITY && OMp[k - 1] > v) { v = OMp[k - 1]; from = FROM_M; }
        if (tr[3] > -INFINITY && OIp[k - 1] > v) { v = OIp[k - 1]; from = FROM_I; }
        if (tr[5] > -INFINITY && ODp[k - 1] > v) { v = ODp[k - 1]; from = FROM_D; }
      }
      OMc[k] = pm[k - 1] + v;
      t[3 * k + 0] = (uint8_t)from;
      OIc[k] = -INFINITY;
      t[3 * k + 1] = FROM_M;
      if (k < M && r > 0) {
        const double *tr = p->tr + (k - 1) * 7;
        double u = -INFINITY;
        int f = FROM_M;
        if (tr[1] > -INFINITY && OMp[k] > u) { u = OMp[k]; f = FROM_M; }
        if (tr[4] > -INFINITY && OIp[k] > u) { u = OIp[k]; f = FROM_I; }
        if (u > -INFINITY) OIc[k] = pi[k - 1] + u;
        t[3 * k + 1] = (uint8_t)f;
      }
    }
    ODc[1] = -INFINITY;
    t[3 * 1 + 2] = FROM_M;
    for (int k = 2; k <= M; k++) {
      const double *tr = p->tr + (k - 2) * 7;
      double u = -INFINITY;
      int f = FROM_M;
      if (tr[2] > -INFINITY && OMc[k - 1] > u) { u = OMc[k - 1]; f = FROM_M; }
      if (tr[6] > -INFINITY && ODc[k - 1] > u) { u = ODc[k - 1]; f = FROM_D; }
      ODc[k] = u;
      t[3 * k + 2] = (uint8_t)f;
    }
    for (int k = 1; k <= M; k++) {
      double sc = OMc[k] + (G[R] - G[r + 1]);
      if (sc > best) { best = sc; bi = r; bk = k; }
    }
    double *tmp;
    tmp = OMp; OMp = OMc; OMc = tmp;
    tmp = OIp; OIp = OIc; OIc = tmp;
    tmp = ODp; ODp = ODc; ODc = tmp;
  }
  if (bi >= 0) {
    for (int r = 0; r < R; r++) code[r] = 0;
    int r = bi, k = bk, st = FROM_M;
    abk[1] = s + bi;
    abk[3] = bk;
    for (;;) {
      const uint8_t *t = tb + (size_t)r * W * 3;
      if (st == FROM_M) {
        code[r] = (int16_t)k;
        const int f = t[3 * k + 0];
        if (f == FROM_B) { abk[0] = s + r; abk[2] = k; break; }
        r--; k--; st = f;
      } else if (st == FROM_I) {
        code[r] = (int16_t)(-k);
        const int f = t[3 * k + 1];
        r--; st = f;
      } else {  /* D_k, same row: predecessor M_{k-1} or D_{k-1} */
        const int f = t[3 * k + 2];
        k--; st = f;
      }
    }
  }
  free(OMp); free(OIp); free(ODp); free(OMc); free(OIc); free(ODc); free(tb); free(G);
  return best;
}

/*
 * Score of a given alignment of region [s, e] under the objective of
 * orc_oa_align, and whether it is a valid path: codes 0 outside one
 * contiguous aligned range [a, b], which starts and ends in a match state;
 * consecutive aligned residues follow M_k -> M_{k+1} (MM), M_k -> I_k (MI),
 * I_k -> I_k (II), I_k -> M_{k+1} (IM), or M_k -> D_{k+1} .. D_{k'-1} ->
 * M_{k'} (MD, DD.., DM), each transition of non-zero probability.
 * *valid receives 1 or 0.
 */
double orc_oa_path_score(const orc_profile *p, int L, const double *pcore, const double *pM, const double *pI,
                         int s, int e, const int16_t *code, int *valid) {
  const int M = p->M;
  *valid = 0;
  if (s < 1 || e > L || s > e) return -INFINITY;
  const int R = e - s + 1;
  int a = -1, b = -1;
  for (int r = 0; r < R; r++)
    if (code[r] != 0) { if (a < 0) a = r; b = r; }
  if (a < 0) return -INFINITY;
  double sc = 0.0;
  for (int r = 0; r < R; r++) {
    const int i = s + r, c = code[r];
    if (r < a || r > b) { sc += 1.0 - pcore[i - 1]; continue; }
    if (c == 0 || c > M || c < -(M - 1)) return -INFINITY;
    sc += c > 0 ? pM[(size_t)(i - 1) * M + (c - 1)] : pI[(size_t)(i - 1) * M + (-c - 1)];
  }
  if (code[a] <= 0 || code[b] <= 0) return -INFINITY;
  for (int r = a; r < b; r++) {
    const int c0 = code[r], c1 = code[r + 1];
    if (c0 > 0 && c1 > 0) {            /* M_k -> M_k' */
      const int k = c0, k2 = c1;
      if (k2 <= k) return -INFINITY;
      const double *t = p->tr + (k - 1) * 7;
      if (k2 == k + 1) {
        if (t[0] == -INFINITY) return -INFINITY;
      } else {
        if (t[2] == -INFINITY) return -INFINITY;                          /* M_k -> D_{k+1} */
        for (int j = k + 1; j < k2 - 1; j++)
          if (p->tr[(j - 1) * 7 + 6] == -INFINITY) return -INFINITY;     /* D_j -> D_{j+1} */
        if (p->tr[(k2 - 2) * 7 + 5] == -INFINITY) return -INFINITY;      /* D_{k2-1} -> M_k2 */
      }
    } else if (c0 > 0 && c1 < 0) {     /* M_k -> I_k */
      if (-c1 != c0 || p->tr[(c0 - 1) * 7 + 1] == -INFINITY) return -INFINITY;
    } else if (c0 < 0 && c1 < 0) {     /* I_k -> I_k */
      if (c1 != c0 || p->tr[(-c0 - 1) * 7 + 4] == -INFINITY) return -INFINITY;
    } else {                           /* I_k -> M_{k+1} */
      if (c1 != -c0 + 1 || p->tr[(-c0 - 1) * 7 + 3] == -INFINITY) return -INFINITY;
    }
  }
  *valid = 1;
  return sc;
}

/* The pipeline without the composition-bias filter. */
int orc_search(const orc_profile *p, const uint8_t *res, const int64_t *off, int64_t n,
               const double *calib, const double *F, int nthreads, int fwd_scaled,
               int16_t *msv, int32_t *vit, double *fwd, uint8_t *flags, double *stage_s) {
  return orc_search_bias(p, res, off, n, calib, F, nthreads, fwd_scaled, 0, msv, vit, fwd, flags, NULL, stage_s);
}
