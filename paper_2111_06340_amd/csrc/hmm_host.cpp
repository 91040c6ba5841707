// Host side of the GPU library: C ABI, argument validation, profile
// quantisation and device table layout, database packing, and the search
// driver.  The scoring model is the one stated in include/hmmgpu.h.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <numeric>
#include <string>
#include <vector>

#include "hmm_internal.h"

using namespace hmmgpu;

namespace {

thread_local std::string g_last_error;

int fail(int code, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

int fail_hip(hipError_t e, const char *what) {
  return fail(HMM_EDEVICE, "%s: %s", what, hipGetErrorString(e));
}

#define HIP_TRY(expr, what)                    \
  do {                                         \
    hipError_t e_ = (expr);                    \
    if (e_ != hipSuccess) return fail_hip(e_, what); \
  } while (0)

// ---------------------------------------------------------------- scores
//
// Quantised score systems (fp64 on the host, rounding q(x) = floor(x + 1/2)):
//   MSV, 1/3-bit units:   sc8 = q(3/ln2 * ln(e/f)); BIAS8 = clamp(-min sc8, 0, 255);
//                         COST8 = clamp(BIAS8 - sc8, 0, 255); ENTRY8 = q(-3/ln2 * ENTRY);
//                         EXIT8 = q(3/ln2 * ln 2); MOVE8(L) = clamp(q(-3/ln2 * MOVE(L)), 0, 255)
//   Viterbi, 1/500 bits:  score16 = sat16(q(500/ln2 * score)); t = 0 -> -32768
// with ENTRY = ln(2/(M(M+1))), MOVE(L) = ln(3/(L+3)), LOOP(L) = ln(L/(L+3)).
// The host evaluates each expression in the same fp64 order so that the
// integer tables are reproducible.

constexpr double kS8 = 3.0 / M_LN2;
constexpr double kS16 = 500.0 / M_LN2;

long q_round(double x) { return (long)std::floor(x + 0.5); }
long clampl(long v, long lo, long hi) { return v < lo ? lo : (v > hi ? hi : v); }

double ln_entry(int M) { return std::log(2.0 / ((double)M * ((double)M + 1.0))); }
double ln_move(int L) { return std::log(3.0 / ((double)L + 3.0)); }
double ln_loop(int L) { return std::log((double)L / ((double)L + 3.0)); }
double null_score(int L) {
  return (double)L * std::log((double)L / ((double)L + 1.0)) + std::log(1.0 / ((double)L + 1.0));
}
int move8_of(int L) { return (int)clampl(q_round(-kS8 * ln_move(L)), 0, 255); }
int move16_of(int L) { return (int)clampl(q_round(kS16 * ln_move(L)), -32768, 32767); }

int instantiated_q8(int q) {
  static const int qs[] = {1, 2, 3, 4, 5, 6, 7, 8, 10, 12, 14, 16, 20, 24};
  for (int v : qs)
    if (v >= q) return v;
  return -1;
}
int instantiated_q32(int q) {
  static const int qs[] = {1, 2, 3, 4, 5, 6, 8, 10, 12, 14, 16, 20, 24, 28, 32, 40, 48};
  for (int v : qs)
    if (v >= q) return v;
  return -1;
}

std::atomic<uint64_t> g_profile_serial{1};

// Device memory the decoding scratch of one database may take.
constexpr size_t kDecodeScratchMax = (size_t)16 << 30;

}  // namespace

struct hmm_profile {
  int M = 0;
  uint64_t serial = 0;
  double mu_msv = 0, mu_vit = 0, tau = 0;
  // host copies
  int bias8 = 0, entry8 = 0, exit8 = 0, entry16 = 0, ej16 = 0;
  std::vector<uint8_t> cost8;
  std::vector<int16_t> msc16, isc16, t16;
  int s_max = 0;  // largest emission score (int16 units, >= 0)
  DevProfile dev{};
  void *dmem = nullptr;  // one device allocation holding every table
};

// Packed residues and index arrays of a database, shared by its handles.
struct hmm_db_data {
  void *dmem = nullptr;
  std::atomic<int> refs{1};
};

struct hmm_db {
  int64_t n = 0, n_res = 0;
  int32_t max_len = 0;
  hmm_db_data *data = nullptr;  // shared with the handles made by hmm_db_share
  void *smem = nullptr;         // this handle's search scratch
  DevDb dev{};
  LenParams *h_lp = nullptr;  // pinned staging of the per-length table
  LenParams *d_lp = nullptr;
  // cache key of the per-length table
  uint64_t lp_serial = 0;
  double lp_F[3] = {-1, -1, -1};
  hipEvent_t done = nullptr;   // completion of the latest search
  bool searched = false;
  // Streams and events of the pipelined cascade (see SearchSync), and the
  // chunking: `chunks` contiguous ranges of the sorted targets, range k =
  // [chunk_at[chunks][k], chunk_at[chunks][k+1]), of about equal residues.
  SearchSync sync;
  int chunks = 1;
  // the stages after MSV: 1 staged kernels, 2 one fused kernel where the
  // profile has an instance, 3 fused when the Viterbi cutoff passes every
  // target (hmm_db_fused_tail)
  int fused_tail = 3;
  int64_t chunk_at[kMaxChunks + 1][kMaxChunks + 1] = {};
  // posterior-decoding scratch (allocated by the first hmm_decode)
  void *dec_mem = nullptr;
  size_t dec_bytes = 0;
  // stage timing ring (profiling hook)
  std::vector<hipEvent_t> tev;  // capacity * 5
  int32_t tcap = 0;
  int64_t trec = 0;             // searches recorded since the last read
};

static void release_sync(hmm_db *db);

namespace {

// ---------------------------------------------------------------- checks

int check_distribution(const double *p, int n, bool strictly_positive, const char *what, int row) {
  double s = 0.0;
  for (int i = 0; i < n; i++) {
    if (!(p[i] >= 0.0) || !std::isfinite(p[i]))
      return fail(HMM_EINVAL, "%s row %d: entry %d is negative or not finite", what, row, i);
    if (strictly_positive && !(p[i] > 0.0))
      return fail(HMM_EINVAL, "%s row %d: entry %d must be > 0", what, row, i);
    s += p[i];
  }
  if (std::fabs(s - 1.0) > 1e-6) return fail(HMM_EINVAL, "%s row %d sums to %.9f, not 1", what, row, s);
  return HMM_OK;
}

int validate_desc(const hmm_profile_desc *d) {
  if (!d) return fail(HMM_EINVAL, "profile descriptor is NULL");
  if (d->M < 1) return fail(HMM_EINVAL, "M = %d; need M >= 1", d->M);
  if (d->M > HMM_MAX_M) return fail(HMM_ERANGE, "M = %d exceeds HMM_MAX_M = %d", d->M, HMM_MAX_M);
  if (!d->bg || !d->match) return fail(HMM_EINVAL, "bg or match is NULL");
  if (d->M > 1 && (!d->insert || !d->trans)) return fail(HMM_EINVAL, "insert or trans is NULL with M > 1");
  if (!std::isfinite(d->mu_msv) || !std::isfinite(d->mu_vit) || !std::isfinite(d->tau))
    return fail(HMM_EINVAL, "calibration values must be finite");
  int rc;
  if ((rc = check_distribution(d->bg, kAlpha, true, "bg", 0))) return rc;
  for (int k = 0; k < d->M; k++)
    if ((rc = check_distribution(d->match + (size_t)k * kAlpha, kAlpha, true, "match", k))) return rc;
  for (int k = 0; k + 1 < d->M; k++) {
    if ((rc = check_distribution(d->insert + (size_t)k * kAlpha, kAlpha, false, "insert", k))) return rc;
    const double *t = d->trans + (size_t)k * 7;
    if ((rc = check_distribution(t, 3, false, "trans MM/MI/MD", k))) return rc;
    if ((rc = check_distribution(t + 3, 2, false, "trans IM/II", k))) return rc;
    if ((rc = check_distribution(t + 5, 2, false, "trans DM/DD", k))) return rc;
  }
  return HMM_OK;
}

// ---------------------------------------------------------------- layout

// Packed 16-bit layout of the MSV and int16 Viterbi kernels: the 128 slots
// of a wave are (lane l, half h) -> slot 2l+h, and slot s holds cells
// s*Q + q in its Q vectors, so a cell's left neighbour lives in the same
// slot one vector earlier, except for vector 0 (previous slot, vector Q-1).
inline size_t pk_index(int q, int lane) { return (size_t)q * kWave + lane; }
inline int pk_cell(int Q, int q, int lane, int half) { return (2 * lane + half) * Q + q; }

// 32-bit layout of the rescore and Forward kernels: slot = lane, cell l*Q + q.
inline int w_cell(int Q, int q, int lane) { return lane * Q + q; }

uint32_t pack16(int lo, int hi) { return (uint32_t)(uint16_t)lo | ((uint32_t)(uint16_t)hi << 16); }

// IEEE binary16 encoding of an integer with |v| <= 2048 (exact).
uint16_t half_of_int(int v) {
  if (v == 0) return 0;
  const uint16_t sign = v < 0 ? 0x8000 : 0;
  const unsigned a = (unsigned)(v < 0 ? -v : v);
  const int e = 31 - __builtin_clz(a);                       // a = 2^e * 1.m
  const unsigned m = e <= 10 ? (a << (10 - e)) & 0x3ffu : (a >> (e - 10)) & 0x3ffu;
  return (uint16_t)(sign | ((unsigned)(e + 15) << 10) | m);
}

// Host quantisation of a validated descriptor into p's host tables.
void quantize(const hmm_profile_desc *d, hmm_profile *p) {
  const int M = d->M;
  p->M = M;
  p->serial = g_profile_serial.fetch_add(1);
  p->mu_msv = d->mu_msv;
  p->mu_vit = d->mu_vit;
  p->tau = d->tau;
  const double entry = ln_entry(M);
  std::vector<long> sc8((size_t)M * kAlpha);
  long min8 = 0;
  for (int k = 0; k < M; k++)
    for (int a = 0; a < kAlpha; a++) {
      long v = q_round(kS8 * std::log(d->match[(size_t)k * kAlpha + a] / d->bg[a]));
      sc8[(size_t)k * kAlpha + a] = v;
      if ((k == 0 && a == 0) || v < min8) min8 = v;
    }
  p->bias8 = (int)clampl(-min8, 0, 255);
  p->cost8.resize((size_t)M * kAlpha);
  for (size_t i = 0; i < sc8.size(); i++) p->cost8[i] = (uint8_t)clampl(p->bias8 - sc8[i], 0, 255);
  p->entry8 = (int)clampl(q_round(-kS8 * entry), 0, 255);
  p->exit8 = (int)clampl(q_round(kS8 * std::log(2.0)), 0, 255);
  p->msc16.resize((size_t)M * kAlpha);
  for (int k = 0; k < M; k++)
    for (int a = 0; a < kAlpha; a++)
      p->msc16[(size_t)k * kAlpha + a] = (int16_t)clampl(
          q_round(kS16 * std::log(d->match[(size_t)k * kAlpha + a] / d->bg[a])), -32768, 32767);
  p->isc16.resize((size_t)std::max(M - 1, 0) * kAlpha);
  p->t16.resize((size_t)std::max(M - 1, 0) * 7);
  for (int k = 0; k + 1 < M; k++) {
    for (int a = 0; a < kAlpha; a++) {
      double e = d->insert[(size_t)k * kAlpha + a];
      // a zero insert probability has score -inf: saturate at the floor
      p->isc16[(size_t)k * kAlpha + a] =
          e > 0.0 ? (int16_t)clampl(q_round(kS16 * std::log(e / d->bg[a])), -32768, 32767) : (int16_t)kNeg16;
    }
    for (int t = 0; t < 7; t++) {
      double v = d->trans[(size_t)k * 7 + t];
      p->t16[(size_t)k * 7 + t] =
          v > 0.0 ? (int16_t)clampl(q_round(kS16 * std::log(v)), -32768, 32767) : (int16_t)kNeg16;
    }
  }
  p->s_max = 0;
  for (int16_t v : p->msc16) p->s_max = std::max(p->s_max, (int)v);
  for (int16_t v : p->isc16) p->s_max = std::max(p->s_max, (int)v);
  p->entry16 = (int)clampl(q_round(kS16 * entry), -32768, 32767);
  p->ej16 = (int)clampl(q_round(kS16 * std::log(0.5)), -32768, 32767);

}

}  // namespace

extern "C" {

const char *hmm_strerror(int status) {
  switch (status) {
    case HMM_OK: return "success";
    case HMM_EINVAL: return "invalid argument";
    case HMM_ERANGE: return "size out of range";
    case HMM_ENOMEM: return "out of memory";
    case HMM_EDEVICE: return "GPU runtime error";
    default: return "unknown status";
  }
}

const char *hmm_last_error(void) { return g_last_error.c_str(); }

int hmm_profile_upload(const hmm_profile_desc *d, hmm_stream stream, hmm_profile **out) {
  if (!out) return fail(HMM_EINVAL, "out is NULL");
  *out = nullptr;
  int rc = validate_desc(d);
  if (rc) return rc;
  const int M = d->M;
  hmm_profile *p = new (std::nothrow) hmm_profile();
  if (!p) return fail(HMM_ENOMEM, "host allocation failed");
  quantize(d, p);

  // ---- device layouts
  const int Q8 = instantiated_q8(q8_of(M));
  const int Q32 = instantiated_q32(q32_of(M));
  // MSV: diagonal layout when M + 1 cells fit a kernel instance of at most
  // kMaxQDiag vectors per lane (it needs one padding cell), else striped.
  const bool msv_diag = q8_of(M + 1) <= kMaxQDiag;
  const int Qm = msv_diag ? instantiated_q8(q8_of(M + 1)) : instantiated_q8(std::max(q8_of(M), kMaxQDiag));
  if (Q8 < 0 || Q32 < 0 || Qm < 0) {
    delete p;
    return fail(HMM_ERANGE, "M = %d has no kernel instance", M);
  }
  const size_t n_msv = (size_t)kAlpha * Qm * kWave * (msv_diag ? 2 : 1);  // dwords
  const size_t n_vemit = (size_t)kAlpha * 2 * Q8 * kWave;
  const size_t n_vtr = (size_t)TR_N * Q8 * kWave;
  const size_t n_w32emit = (size_t)kAlpha * 2 * Q32 * kWave;
  const size_t n_w32tr = (size_t)TR_N * Q32 * kWave;
  const size_t n_ftr = (size_t)(TR_N + 3) * Q32 * kWave;
  const size_t total = n_msv + n_vemit + n_vtr + n_w32emit + n_w32tr + n_w32emit + n_ftr;
  std::vector<uint32_t> h(total, 0);
  uint32_t *h_msv = h.data();
  uint32_t *h_vemit = h_msv + n_msv;
  uint32_t *h_vtr = h_vemit + n_vemit;
  int32_t *h_w32emit = (int32_t *)(h_vtr + n_vtr);
  int32_t *h_w32tr = h_w32emit + n_w32emit;
  float *h_femit = (float *)(h_w32tr + n_w32tr);
  float *h_ftr = h_femit + n_w32emit;

  auto t16 = [&](int node, int which) -> int {  // node 1..M-1
    return p->t16[(size_t)(node - 1) * 7 + which];
  };
  // transition of plane `tr` into/at cell c (0-based; node c+1); INT_MIN = structural
  const int kNone = INT32_MIN;
  auto tr_cell = [&](int tr, int c) -> int {
    if (c >= M) return kNone;
    switch (tr) {
      case TR_MMIN: return c >= 1 ? t16(c, 0) : kNone;
      case TR_IMIN: return c >= 1 ? t16(c, 3) : kNone;
      case TR_DMIN: return c >= 1 ? t16(c, 5) : kNone;
      case TR_MDIN: return c >= 1 ? t16(c, 2) : kNone;
      case TR_DDIN: return c >= 1 ? t16(c, 6) : kNone;
      case TR_MI: return c + 1 < M ? t16(c + 1, 1) : kNone;
      case TR_II: return c + 1 < M ? t16(c + 1, 4) : kNone;
    }
    return kNone;
  };
  auto tr_prob = [&](int tr, int c) -> double {
    if (c >= M) return 0.0;
    auto t = [&](int node, int which) { return d->trans[(size_t)(node - 1) * 7 + which]; };
    switch (tr) {
      case TR_MMIN: return c >= 1 ? t(c, 0) : 0.0;
      case TR_IMIN: return c >= 1 ? t(c, 3) : 0.0;
      case TR_DMIN: return c >= 1 ? t(c, 5) : 0.0;
      case TR_MDIN: return c >= 1 ? t(c, 2) : 0.0;
      case TR_DDIN: return c >= 1 ? t(c, 6) : 0.0;
      case TR_MI: return c + 1 < M ? t(c + 1, 1) : 0.0;
      case TR_II: return c + 1 < M ? t(c + 1, 4) : 0.0;
    }
    return 0.0;
  };
  auto msc_cell = [&](int c, int a) -> int { return c < M ? p->msc16[(size_t)c * kAlpha + a] : kNone; };
  auto isc_cell = [&](int c, int a) -> int { return c + 1 < M ? p->isc16[(size_t)c * kAlpha + a] : kNone; };
  auto lo16 = [](int v) { return v == INT32_MIN ? kNeg16 : v; };

  // MSV scores E = BIAS8 - COST8 as fp16 (exact small integers); padding -1024.
  auto msv_e = [&](int c, int a) -> uint16_t {
    return half_of_int(c < M ? p->bias8 - (int)p->cost8[(size_t)c * kAlpha + a] : -1024);
  };
  if (msv_diag) {
    const int P = 2 * Qm * kWave;
    for (int a = 0; a < kAlpha; a++)
      for (int c = 0; c < P; c++)
        h_msv[(size_t)a * P + c] = (uint32_t)msv_e(c, a) | ((uint32_t)msv_e((c + P / 2) % P, a) << 16);
  } else {
    for (int a = 0; a < kAlpha; a++)
      for (int q = 0; q < Qm; q++)
        for (int l = 0; l < kWave; l++)
          h_msv[(size_t)a * Qm * kWave + pk_index(q, l)] =
              (uint32_t)msv_e(pk_cell(Qm, q, l, 0), a) | ((uint32_t)msv_e(pk_cell(Qm, q, l, 1), a) << 16);
  }
  for (int a = 0; a < kAlpha; a++)
    for (int q = 0; q < Q8; q++)
      for (int l = 0; l < kWave; l++) {
        int c0 = pk_cell(Q8, q, l, 0), c1 = pk_cell(Q8, q, l, 1);
        h_vemit[((size_t)a * 2 + 0) * Q8 * kWave + pk_index(q, l)] =
            pack16(lo16(msc_cell(c0, a)), lo16(msc_cell(c1, a)));
        h_vemit[((size_t)a * 2 + 1) * Q8 * kWave + pk_index(q, l)] =
            pack16(lo16(isc_cell(c0, a)), lo16(isc_cell(c1, a)));
      }
  for (int tr = 0; tr < TR_N; tr++)
    for (int q = 0; q < Q8; q++)
      for (int l = 0; l < kWave; l++)
        h_vtr[(size_t)tr * Q8 * kWave + pk_index(q, l)] =
            pack16(lo16(tr_cell(tr, pk_cell(Q8, q, l, 0))), lo16(tr_cell(tr, pk_cell(Q8, q, l, 1))));
  auto w32 = [&](int v) { return v == INT32_MIN ? kNeg32 : v; };
  for (int a = 0; a < kAlpha; a++)
    for (int q = 0; q < Q32; q++)
      for (int l = 0; l < kWave; l++) {
        int c = w_cell(Q32, q, l);
        size_t im = ((size_t)a * 2 + 0) * Q32 * kWave + pk_index(q, l);
        size_t ii = ((size_t)a * 2 + 1) * Q32 * kWave + pk_index(q, l);
        h_w32emit[im] = w32(msc_cell(c, a));
        h_w32emit[ii] = w32(isc_cell(c, a));
        h_femit[im] = c < M ? (float)(d->match[(size_t)c * kAlpha + a] / d->bg[a]) : 0.0f;
        h_femit[ii] = c + 1 < M ? (float)(d->insert[(size_t)c * kAlpha + a] / d->bg[a]) : 0.0f;
      }
  for (int tr = 0; tr < TR_N; tr++)
    for (int q = 0; q < Q32; q++)
      for (int l = 0; l < kWave; l++) {
        int c = w_cell(Q32, q, l);
        h_w32tr[(size_t)tr * Q32 * kWave + pk_index(q, l)] = w32(tr_cell(tr, c));
        h_ftr[(size_t)tr * Q32 * kWave + pk_index(q, l)] = (float)tr_prob(tr, c);
      }
  // D-chain products inside each slot.  Forward (cell k-1 -> k):
  // prod_{j<=q} DDin(cell l*Q+j).  Backward (cell k+1 -> k):
  // prod_{j=q+1}^{Q} DDin(cell l*Q+j), whose last factor is the next slot's
  // first cell (0 past the last slot).
  for (int l = 0; l < kWave; l++) {
    double acc = 1.0;
    for (int q = 0; q < Q32; q++) {
      acc *= tr_prob(TR_DDIN, w_cell(Q32, q, l));
      h_ftr[(size_t)TR_PRE * Q32 * kWave + pk_index(q, l)] = (float)acc;
    }
    acc = l + 1 < kWave ? tr_prob(TR_DDIN, w_cell(Q32, 0, l + 1)) : 0.0;
    for (int q = Q32 - 1; q >= 0; q--) {
      h_ftr[(size_t)TR_SUF * Q32 * kWave + pk_index(q, l)] = (float)acc;
      acc *= tr_prob(TR_DDIN, w_cell(Q32, q, l));
    }
  }

  // Exit weights.  A row's delete cells are sums over the same row's match
  // cells: D_c = sum_{j<c} M_j MDIN(j+1) DDIN(j+2) ... DDIN(c), so the row's
  // E = sum_c (M_c + D_c) = sum_j M_j g_j with
  //   g_j = 1 + MDIN(j+1) S_{j+1},  S_k = 1 + DDIN(k+1) S_{k+1},
  // the total probability of leaving M_j for E directly or through the
  // delete states it reaches (zero transitions past the last node end the
  // sums).  fp64, cells P-1 down to 0.
  {
    const int P32 = Q32 * kWave;
    double S = 1.0;   // S_{c+1} while cell c is visited
    for (int c = P32 - 1; c >= 0; c--) {
      const double g = 1.0 + (c + 1 < P32 ? tr_prob(TR_MDIN, c + 1) * S : 0.0);
      h_ftr[(size_t)TR_EXIT * Q32 * kWave + pk_index(c % Q32, c / Q32)] = c < M ? (float)g : 0.0f;
      S = 1.0 + (c + 1 < P32 ? tr_prob(TR_DDIN, c + 1) * S : 0.0);
    }
  }

  hipError_t e = hipMalloc(&p->dmem, total * sizeof(uint32_t));
  if (e != hipSuccess) {
    delete p;
    return e == hipErrorOutOfMemory ? fail(HMM_ENOMEM, "device allocation of %zu bytes failed", total * 4)
                                    : fail_hip(e, "hipMalloc");
  }
  e = hipMemcpyAsync(p->dmem, h.data(), total * sizeof(uint32_t), hipMemcpyHostToDevice, (hipStream_t)stream);
  if (e == hipSuccess) e = hipStreamSynchronize((hipStream_t)stream);
  if (e != hipSuccess) {
    (void)hipFree(p->dmem);
    delete p;
    return fail_hip(e, "profile upload");
  }
  const uint32_t *base = (const uint32_t *)p->dmem;
  DevProfile &dv = p->dev;
  dv.M = M;
  dv.Q8 = Q8;
  dv.Q32 = Q32;
  dv.Qm = Qm;
  dv.msv_diag = msv_diag ? 1 : 0;
  dv.bias8 = p->bias8;
  dv.entry8 = p->entry8;
  dv.exit8 = p->exit8;
  dv.entry16 = p->entry16;
  dv.ej16 = p->ej16;
  dv.dm_max16 = kNeg16;
  dv.dm_max32 = kNeg32;
  for (int c = 1; c < M; c++) {
    dv.dm_max16 = std::max(dv.dm_max16, lo16(tr_cell(TR_DMIN, c)));
    dv.dm_max32 = std::max(dv.dm_max32, w32(tr_cell(TR_DMIN, c)));
  }
  dv.entry_p = (float)(2.0 / ((double)M * ((double)M + 1.0)));
  for (int a = 0; a < kAlpha; a++) {
    double m = 0.0;
    for (int k = 0; k < M; k++) m += d->match[(size_t)k * kAlpha + a];
    dv.bias_r[a] = (float)(m / (double)M / d->bg[a]);
  }
  dv.msv = base;
  dv.vit_emit = base + n_msv;
  dv.vit_tr = dv.vit_emit + n_vemit;
  dv.v32_emit = (const int32_t *)(dv.vit_tr + n_vtr);
  dv.v32_tr = dv.v32_emit + n_w32emit;
  dv.f_emit = (const float *)(dv.v32_tr + n_w32tr);
  dv.f_tr = dv.f_emit + n_w32emit;
  *out = p;
  return HMM_OK;
}

int hmm_profile_free(hmm_profile *p) {
  if (!p) return HMM_OK;
  hipError_t e = p->dmem ? hipFree(p->dmem) : hipSuccess;
  delete p;
  if (e != hipSuccess) return fail_hip(e, "hipFree(profile)");
  return HMM_OK;
}

int hmm_debug_tables(const hmm_profile_desc *d, int32_t *scalars, uint8_t *cost8, int16_t *msc16,
                     int16_t *isc16, int16_t *t16) {
  if (!scalars) return fail(HMM_EINVAL, "scalars is NULL");
  int rc = validate_desc(d);
  if (rc) return rc;
  hmm_profile p;
  quantize(d, &p);
  scalars[0] = p.bias8;
  scalars[1] = p.entry8;
  scalars[2] = p.exit8;
  scalars[3] = p.entry16;
  scalars[4] = p.ej16;
  scalars[5] = p.M;
  scalars[6] = instantiated_q8(q8_of(p.M));
  scalars[7] = instantiated_q32(q32_of(p.M));
  if (cost8) memcpy(cost8, p.cost8.data(), p.cost8.size());
  if (msc16) memcpy(msc16, p.msc16.data(), p.msc16.size() * 2);
  if (isc16) memcpy(isc16, p.isc16.data(), p.isc16.size() * 2);
  if (t16) memcpy(t16, p.t16.data(), p.t16.size() * 2);
  return HMM_OK;
}

}  // extern "C"

namespace {

// Per-length parameters: the cutoffs are the smallest integer scores whose
// bit score exceeds the P-value cutoff (slope ln 2 per bit):
//   MSV:     Gumbel, x1 = mu_msv - ln(-ln(1 - F1)) / ln 2
//            THR8  = floor(BASE8 + S8 * (x1 ln2 + NULL(L) + 3)) + 1, in [0, 256]
//   Viterbi: Gumbel, x2 = mu_vit - ln(-ln(1 - F2)) / ln 2
//            THR16 = floor(S16 * (x2 ln2 + NULL(L) + 3)) + 1
//   Forward: exponential tail, pass when fwd > (tau - ln(F3)/ln 2) ln2 + NULL(L)
// (the 3 nats stand for the N/C/J loop scores that the integer filters omit).
void length_params(const hmm_profile *p, const hmm_thresholds *t, int L, LenParams *lp, double *f64) {
  const double nul = null_score(L);
  lp->move8 = move8_of(L);
  lp->move16 = move16_of(L);
  if (t->F1 >= 1.0) {
    lp->thr8 = 0;
  } else {
    double x1 = p->mu_msv - std::log(-std::log(1.0 - t->F1)) / M_LN2;
    double y = std::floor(kBase8 + kS8 * (x1 * M_LN2 + nul + 3.0)) + 1.0;
    lp->thr8 = (int32_t)(y < 0.0 ? 0.0 : (y > 256.0 ? 256.0 : y));
  }
  if (t->F2 >= 1.0) {
    lp->thr16 = INT32_MIN;
  } else {
    double x2 = p->mu_vit - std::log(-std::log(1.0 - t->F2)) / M_LN2;
    double y = std::floor(kS16 * (x2 * M_LN2 + nul + 3.0)) + 1.0;
    lp->thr16 = (int32_t)(y < -2147483647.0 ? -2147483647.0 : (y > 2147483647.0 ? 2147483647.0 : y));
  }
  double fthr = t->F3 >= 1.0 ? -INFINITY : (p->tau - std::log(t->F3) / M_LN2) * M_LN2 + nul;
  lp->loop_p = (float)((double)L / ((double)L + 3.0));
  lp->move_p = (float)(3.0 / ((double)L + 3.0));
  lp->fthr = (float)fthr;
  lp->pad = 0.0f;
  if (f64) {
    f64[0] = ln_loop(L);
    f64[1] = ln_move(L);
    f64[2] = nul;
    f64[3] = fthr;
  }
}

}  // namespace

// The search scratch of one database handle (flags, survivor lists,
// counters, per-length table), its pinned staging of that table, and the
// streams and events that order its searches.
static int attach_scratch(hmm_db *db) {
  auto al = [](size_t v) { return (v + 255) / 256 * 256; };
  const size_t n = (size_t)db->n;
  const size_t sz_u8 = al(n + 1), sz_i32 = al(n * 4 + 4);
  const size_t sz_lp = al(sizeof(LenParams) * ((size_t)db->max_len + 1));
  const size_t sz_i16 = al(n * 2 + 2);
  const size_t o_flags = 0, o_msv = o_flags + sz_u8, o_lv = o_msv + sz_i16, o_lo = o_lv + sz_i32,
               o_lf = o_lo + sz_i32;
  const size_t o_cnt = o_lf + sz_i32, o_lp = o_cnt + al(kMaxChunks * CNT_N * 4), total = o_lp + sz_lp;
  hipError_t e = hipMalloc(&db->smem, total);
  if (e != hipSuccess) {
    db->smem = nullptr;
    return e == hipErrorOutOfMemory ? fail(HMM_ENOMEM, "device allocation of %zu bytes failed", total)
                                    : fail_hip(e, "hipMalloc(db scratch)");
  }
  e = hipMemset(db->smem, 0, total);
  if (e == hipSuccess) e = hipHostMalloc((void **)&db->h_lp, sz_lp, hipHostMallocDefault);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&db->done, hipEventDisableTiming);
  SearchSync &y = db->sync;
  for (int k = 0; k < kMaxChunks && e == hipSuccess; k++) {
    e = hipEventCreateWithFlags(&y.msv_done[k], hipEventDisableTiming);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&y.vit_done[k], hipEventDisableTiming);
  }
  if (e == hipSuccess) e = hipEventCreateWithFlags(&y.aux_done, hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&y.tail_done, hipEventDisableTiming);
  // default priority, like every stream here
  if (e == hipSuccess) e = hipStreamCreateWithFlags(&y.tail, hipStreamNonBlocking);
  if (e == hipSuccess) e = hipStreamCreateWithFlags(&y.aux, hipStreamNonBlocking);
  if (e != hipSuccess) return fail_hip(e, "database scratch");
  uint8_t *b = (uint8_t *)db->smem;
  DevDb &dv = db->dev;
  dv.flags_sorted = b + o_flags;
  dv.msv_sorted = (int16_t *)(b + o_msv);
  dv.list_vit = (int32_t *)(b + o_lv);
  dv.list_ovf = (int32_t *)(b + o_lo);
  dv.list_fwd = (int32_t *)(b + o_lf);
  dv.counters = (int32_t *)(b + o_cnt);
  db->d_lp = (LenParams *)(b + o_lp);
  dv.lp = db->d_lp;
  return HMM_OK;
}

extern "C" {

int hmm_debug_length_params(const hmm_profile_desc *d, const hmm_thresholds *t, int32_t L, int32_t *i32,
                            double *f64) {
  if (!d || !t || !i32 || !f64) return fail(HMM_EINVAL, "NULL argument");
  if (L < 1) return fail(HMM_EINVAL, "L = %d; need L >= 1", L);
  if (!std::isfinite(d->mu_msv) || !std::isfinite(d->mu_vit) || !std::isfinite(d->tau))
    return fail(HMM_EINVAL, "calibration values must be finite");
  hmm_profile p;
  p.mu_msv = d->mu_msv;
  p.mu_vit = d->mu_vit;
  p.tau = d->tau;
  LenParams lp;
  length_params(&p, t, L, &lp, f64);
  i32[0] = lp.move8;
  i32[1] = lp.thr8;
  i32[2] = lp.move16;
  i32[3] = lp.thr16;
  i32[4] = 0;
  i32[5] = 0;
  return HMM_OK;
}

int hmm_db_upload(const uint8_t *residues, const int64_t *offsets, int64_t n, hmm_stream stream,
                  hmm_db **out) {
  if (!out) return fail(HMM_EINVAL, "out is NULL");
  *out = nullptr;
  if (n < 0) return fail(HMM_EINVAL, "n_seqs = %lld", (long long)n);
  if (!offsets) return fail(HMM_EINVAL, "offsets is NULL");
  if (offsets[0] != 0) return fail(HMM_EINVAL, "offsets[0] = %lld, must be 0", (long long)offsets[0]);
  if (n > 0 && !residues) return fail(HMM_EINVAL, "residues is NULL");
  if (n > (int64_t)INT32_MAX) return fail(HMM_ERANGE, "too many sequences");
  int32_t max_len = 0;
  for (int64_t i = 0; i < n; i++) {
    int64_t L = offsets[i + 1] - offsets[i];
    if (L < 1) return fail(HMM_EINVAL, "sequence %lld has length %lld; need >= 1", (long long)i, (long long)L);
    if (L > HMM_MAX_LEN)
      return fail(HMM_ERANGE, "sequence %lld has length %lld > HMM_MAX_LEN", (long long)i, (long long)L);
    max_len = std::max<int32_t>(max_len, (int32_t)L);
  }
  const int64_t n_res = offsets[n];
  for (int64_t j = 0; j < n_res; j++)
    if (residues[j] >= kAlpha)
      return fail(HMM_EINVAL, "residue %lld has code %d; codes are 0..19", (long long)j, residues[j]);

  // stable sort by decreasing length
  std::vector<int32_t> order((size_t)n);
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) {
    return offsets[a + 1] - offsets[a] > offsets[b + 1] - offsets[b];
  });
  std::vector<int64_t> start((size_t)n);
  std::vector<int32_t> len((size_t)n);
  int64_t pos = 0;
  for (int64_t i = 0; i < n; i++) {
    int32_t L = (int32_t)(offsets[order[i] + 1] - offsets[order[i]]);
    start[i] = pos;
    len[i] = L;
    pos += ((int64_t)L + 15) / 16 * 16;
  }
  const int64_t res_bytes = pos + 1024;  // residue streams read at most 255 bytes past a target
  // chunk boundaries for every chunk count: about equal residues per chunk
  int64_t chunk_at[kMaxChunks + 1][kMaxChunks + 1] = {};
  for (int K = 1; K <= kMaxChunks; K++) {
    int64_t acc = 0, i = 0;
    chunk_at[K][0] = 0;
    for (int k = 1; k < K; k++) {
      const int64_t goal = n_res * k / K;
      while (i < n && acc + len[i] <= goal) acc += len[i++];
      chunk_at[K][k] = std::max(i, chunk_at[K][k - 1]);
    }
    chunk_at[K][K] = n;
  }
  auto al = [](size_t v) { return (v + 255) / 256 * 256; };
  const size_t sz_res = al((size_t)res_bytes);
  const size_t sz_start = al((size_t)n * 8 + 8), sz_i32 = al((size_t)n * 4 + 4);
  const size_t total = sz_res + sz_start * 2 + sz_i32 * 3;

  hmm_db *db = new (std::nothrow) hmm_db();
  if (!db) return fail(HMM_ENOMEM, "host allocation failed");
  db->n = n;
  db->n_res = n_res;
  db->max_len = max_len;
  memcpy(db->chunk_at, chunk_at, sizeof chunk_at);
  // One chunk: each MSV kernel fills every CU's LDS, so a chunk's Viterbi
  // runs mostly after the next MSV anyway, and every chunk adds an MSV
  // launch and its drain.  Since the MSV waves take their targets from a
  // work counter (no wave is left with a slow share), the sequential search
  // is the fastest measured: 348M residues, M = 734: 14.34 ms against 14.64
  // for two chunks and 15.17 for three; 707M residues, M = 2500: 111.0 ms
  // against 111.8 for two, 112.9 for three and 113.3 for four.
  db->chunks = 1;
  db->data = new (std::nothrow) hmm_db_data();
  if (!db->data) {
    delete db;
    return fail(HMM_ENOMEM, "host allocation failed");
  }
  uint8_t *stage = nullptr;
  hipError_t e = hipHostMalloc((void **)&stage, total, hipHostMallocDefault);
  if (e != hipSuccess) {
    delete db->data;
    delete db;
    return fail(HMM_ENOMEM, "pinned staging of %zu bytes failed: %s", total, hipGetErrorString(e));
  }
  memset(stage, 0, total);
  size_t off = 0;
  uint8_t *s_res = stage + off;
  const size_t o_res = off;
  off += sz_res;
  const size_t o_start = off;
  int64_t *s_start = (int64_t *)(stage + off);
  off += sz_start;
  const size_t o_len = off;
  int32_t *s_len = (int32_t *)(stage + off);
  off += sz_i32;
  const size_t o_perm = off;
  int32_t *s_perm = (int32_t *)(stage + off);
  off += sz_i32;
  const size_t o_coff = off;
  int64_t *s_coff = (int64_t *)(stage + off);
  off += sz_start;
  const size_t o_iperm = off;
  int32_t *s_iperm = (int32_t *)(stage + off);
  off += sz_i32;
  for (int64_t i = 0; i < n; i++) {
    memcpy(s_res + start[i], residues + offsets[order[i]], (size_t)len[i]);
    s_start[i] = start[i];
    s_len[i] = len[i];
    s_perm[i] = order[i];
    s_coff[i] = offsets[order[i]];
    s_iperm[order[i]] = (int32_t)i;
  }
  e = hipMalloc(&db->data->dmem, total);
  if (e != hipSuccess) {
    (void)hipHostFree(stage);
    delete db->data;
    delete db;
    return e == hipErrorOutOfMemory ? fail(HMM_ENOMEM, "device allocation of %zu bytes failed", total)
                                    : fail_hip(e, "hipMalloc(db)");
  }
  e = hipMemcpyAsync(db->data->dmem, stage, total, hipMemcpyHostToDevice, (hipStream_t)stream);
  if (e == hipSuccess) e = hipStreamSynchronize((hipStream_t)stream);
  (void)hipHostFree(stage);
  if (e != hipSuccess) {
    (void)hipFree(db->data->dmem);
    delete db->data;
    delete db;
    return fail_hip(e, "database upload");
  }
  uint8_t *b = (uint8_t *)db->data->dmem;
  DevDb &dv = db->dev;
  dv.n = n;
  dv.max_len = max_len;
  dv.res = b + o_res;
  dv.start = (const int64_t *)(b + o_start);
  dv.len = (const int32_t *)(b + o_len);
  dv.perm = (const int32_t *)(b + o_perm);
  dv.coff = (const int64_t *)(b + o_coff);
  dv.iperm = (const int32_t *)(b + o_iperm);
  const int rc = attach_scratch(db);
  if (rc != HMM_OK) {
    (void)hmm_db_free(db);
    return rc;
  }
  *out = db;
  return HMM_OK;
}

int hmm_db_share(const hmm_db *src, hmm_db **out) {
  if (!src || !out) return fail(HMM_EINVAL, "NULL db or out");
  *out = nullptr;
  hmm_db *db = new (std::nothrow) hmm_db();
  if (!db) return fail(HMM_ENOMEM, "host allocation failed");
  db->n = src->n;
  db->n_res = src->n_res;
  db->max_len = src->max_len;
  db->data = src->data;
  db->data->refs.fetch_add(1);
  db->chunks = src->chunks;
  db->fused_tail = src->fused_tail;
  memcpy(db->chunk_at, src->chunk_at, sizeof db->chunk_at);
  db->dev = src->dev;   // shared residues and index arrays; attach_scratch replaces the rest
  const int rc = attach_scratch(db);
  if (rc != HMM_OK) {
    (void)hmm_db_free(db);
    return rc;
  }
  *out = db;
  return HMM_OK;
}

static void release_sync(hmm_db *db) {
  SearchSync &y = db->sync;
  if (y.tail) (void)hipStreamDestroy(y.tail);
  if (y.aux) (void)hipStreamDestroy(y.aux);
  for (int k = 0; k < kMaxChunks; k++) {
    if (y.msv_done[k]) (void)hipEventDestroy(y.msv_done[k]);
    if (y.vit_done[k]) (void)hipEventDestroy(y.vit_done[k]);
  }
  if (y.aux_done) (void)hipEventDestroy(y.aux_done);
  if (y.tail_done) (void)hipEventDestroy(y.tail_done);
  if (db->done) (void)hipEventDestroy(db->done);
  db->sync = SearchSync{};
  db->done = nullptr;
}

static void drop_timing(hmm_db *db) {
  for (hipEvent_t ev : db->tev) (void)hipEventDestroy(ev);
  db->tev.clear();
  db->tcap = 0;
  db->trec = 0;
}

int hmm_db_stage_timing(hmm_db *db, int32_t capacity) {
  if (!db || capacity < 0) return fail(HMM_EINVAL, "NULL db or negative capacity");
  if (db->searched) HIP_TRY(hipEventSynchronize(db->done), "hipEventSynchronize");
  drop_timing(db);
  for (int32_t i = 0; i < capacity * 5; i++) {
    hipEvent_t ev;
    hipError_t e = hipEventCreate(&ev);
    if (e != hipSuccess) {
      drop_timing(db);
      return fail_hip(e, "hipEventCreate");
    }
    db->tev.push_back(ev);
  }
  db->tcap = capacity;
  return HMM_OK;
}

int hmm_db_stage_times(hmm_db *db, float *out_ms, int32_t cap, int32_t *n) {
  if (!db || !n || (cap > 0 && !out_ms)) return fail(HMM_EINVAL, "NULL argument");
  *n = 0;
  if (db->tcap <= 0) return HMM_OK;
  if (db->searched) HIP_TRY(hipEventSynchronize(db->done), "hipEventSynchronize");
  const int64_t have = std::min<int64_t>(db->trec, db->tcap);
  const int64_t first = db->trec - have;
  int32_t k = 0;
  for (int64_t i = first; i < db->trec && k < cap; i++, k++) {
    hipEvent_t *ev = &db->tev[(size_t)(i % db->tcap) * 5];
    // ev: search start, MSV end, Viterbi end (fork), rescore end (aux
    // stream), end of Forward and rescore (join)
    HIP_TRY(hipEventElapsedTime(&out_ms[4 * k + 0], ev[0], ev[1]), "hipEventElapsedTime");
    HIP_TRY(hipEventElapsedTime(&out_ms[4 * k + 1], ev[1], ev[2]), "hipEventElapsedTime");
    HIP_TRY(hipEventElapsedTime(&out_ms[4 * k + 2], ev[2], ev[3]), "hipEventElapsedTime");
    HIP_TRY(hipEventElapsedTime(&out_ms[4 * k + 3], ev[2], ev[4]), "hipEventElapsedTime");
  }
  *n = k;
  db->trec = 0;
  return HMM_OK;
}

int hmm_probe_pk16(hmm_stream stream, double *ops_per_s, float *ms) {
  if (!ops_per_s) return fail(HMM_EINVAL, "NULL ops_per_s");
  int dev = 0, ncu = 0;
  HIP_TRY(hipGetDevice(&dev), "hipGetDevice");
  HIP_TRY(hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev), "hipDeviceGetAttribute");
  const int64_t words = (int64_t)2 * (ncu > 0 ? ncu : 256) * 1024;
  void *buf = nullptr;
  hipError_t e = hipMalloc(&buf, (size_t)words * 4);
  if (e != hipSuccess)
    return e == hipErrorOutOfMemory ? fail(HMM_ENOMEM, "probe buffer") : fail_hip(e, "hipMalloc(probe buffer)");
  e = probe_pk16((uint32_t *)buf, words, (hipStream_t)stream, ops_per_s, ms);
  const hipError_t f = hipFree(buf);
  if (e != hipSuccess) return fail_hip(e, "packed 16-bit probe");
  if (f != hipSuccess) return fail_hip(f, "hipFree(probe buffer)");
  return HMM_OK;
}

int hmm_db_free(hmm_db *db) {
  if (!db) return HMM_OK;
  hipError_t e = hipSuccess;
  if (db->searched) e = hipEventSynchronize(db->done);
  drop_timing(db);
  release_sync(db);
  if (db->h_lp) (void)hipHostFree(db->h_lp);
  if (db->dec_mem) (void)hipFree(db->dec_mem);
  hipError_t e2 = db->smem ? hipFree(db->smem) : hipSuccess;
  if (db->data && db->data->refs.fetch_sub(1) == 1) {
    const hipError_t e3 = db->data->dmem ? hipFree(db->data->dmem) : hipSuccess;
    if (e2 == hipSuccess) e2 = e3;
    delete db->data;
  }
  delete db;
  if (e != hipSuccess) return fail_hip(e, "hipEventSynchronize(db)");
  if (e2 != hipSuccess) return fail_hip(e2, "hipFree(db)");
  return HMM_OK;
}

int hmm_db_pipeline(hmm_db *db, int32_t chunks, int32_t *current) {
  if (!db) return fail(HMM_EINVAL, "db is NULL");
  if (chunks < 0 || chunks > kMaxChunks) return fail(HMM_EINVAL, "chunks = %d; need 0..%d", chunks, kMaxChunks);
  if (chunks > 0) db->chunks = chunks;   // searches on a handle are serialised on the GPU
  if (current) *current = db->chunks;
  return HMM_OK;
}

int hmm_db_fused_tail(hmm_db *db, int32_t mode, int32_t *current) {
  if (!db) return fail(HMM_EINVAL, "db is NULL");
  if (mode < 0 || mode > 3) return fail(HMM_EINVAL, "mode = %d; need 0..3", mode);
  if (mode > 0) db->fused_tail = mode;   // searches on a handle are serialised on the GPU
  if (current) *current = db->fused_tail;
  return HMM_OK;
}

int hmm_db_info(const hmm_db *db, int64_t *n_seqs, int64_t *n_residues, int32_t *max_len) {
  if (!db) return fail(HMM_EINVAL, "db is NULL");
  if (n_seqs) *n_seqs = db->n;
  if (n_residues) *n_residues = db->n_res;
  if (max_len) *max_len = db->max_len;
  return HMM_OK;
}

// Whether a search runs its stages after MSV as one kernel (mode of
// hmm_db_fused_tail).  In mode 3 it does when the Viterbi cutoff passes every
// target: then every target that reaches Viterbi also reaches Forward, and a
// wave that takes each through all its stages saves two stage boundaries.
// With a Viterbi filter most targets stop there, and the staged int16
// kernel, at twice the waves per SIMD (the fused kernel's registers are set
// by its Forward), is the faster one.
static int fuse_tail(int mode, const hmm_thresholds &t) { return mode == 2 || (mode == 3 && t.F2 >= 1.0); }

// Every transition score is <= 0 and a path emits at most once per residue,
// so no Viterbi value of a target of length L exceeds L * s_max.  The int32
// rescore is exact while that stays below 2^29 (its delete floor drops
// sums with a structural -2^30 only below that).  With a background whose
// rarest residue has frequency 1.3 %, no emission scores above about 3,100
// units, against the 5,368 allowed for 100,000 residues.
static bool int32_range_ok(const hmm_profile *p, const hmm_db *db) {
  return (int64_t)db->max_len * p->s_max < ((int64_t)1 << 29);
}

int hmm_search(const hmm_profile *p, hmm_db *db, const hmm_thresholds *t, const hmm_results *out,
               hmm_stream stream) {
  if (!p || !db || !t || !out) return fail(HMM_EINVAL, "NULL profile, db, thresholds or results");
  if (std::isnan(t->F1) || std::isnan(t->F2) || std::isnan(t->F3) || !(t->F1 > 0) || !(t->F2 > 0) ||
      !(t->F3 > 0))
    return fail(HMM_EINVAL, "P-value cutoffs must be > 0");
  if (t->bias_filter != 0 && t->bias_filter != 1) return fail(HMM_EINVAL, "bias_filter = %d; need 0 or 1", t->bias_filter);
  if (db->n > 0 && (!out->msv || !out->vit || !out->fwd || !out->flags))
    return fail(HMM_EINVAL, "NULL output buffer");
  if (!int32_range_ok(p, db))
    return fail(HMM_ERANGE, "longest target (%d) times largest emission score (%d) reaches 2^29", db->max_len,
                p->s_max);
  hipStream_t s = (hipStream_t)stream;
  if (db->n == 0) return HMM_OK;
  // serialise searches on this database (scratch and per-length table)
  if (db->searched) HIP_TRY(hipStreamWaitEvent(s, db->done, 0), "hipStreamWaitEvent");
  if (db->lp_serial != p->serial || db->lp_F[0] != t->F1 || db->lp_F[1] != t->F2 || db->lp_F[2] != t->F3) {
    if (db->searched) HIP_TRY(hipEventSynchronize(db->done), "hipEventSynchronize");
    for (int L = 0; L <= db->max_len; L++) length_params(p, t, L < 1 ? 1 : L, &db->h_lp[L], nullptr);
    HIP_TRY(hipMemcpyAsync(db->d_lp, db->h_lp, sizeof(LenParams) * ((size_t)db->max_len + 1),
                           hipMemcpyHostToDevice, s),
            "hipMemcpyAsync(length table)");
    db->lp_serial = p->serial;
    db->lp_F[0] = t->F1;
    db->lp_F[1] = t->F2;
    db->lp_F[2] = t->F3;
  }
  DevOut o{out->msv,  out->vit,       out->fwd, out->flags, out->counts,
           out->bias, t->bias_filter, fuse_tail(db->fused_tail, *t)};
  hipEvent_t *ev = nullptr;
  if (db->tcap > 0) ev = &db->tev[(size_t)(db->trec++ % db->tcap) * 5];
  DevDb chunk[kMaxChunks];
  const int K = db->chunks;
  for (int k = 0; k < K; k++) chunk[k] = chunk_of(db->dev, db->chunk_at[K][k], db->chunk_at[K][k + 1], k);
  HIP_TRY(launch_search(p->dev, chunk, K, o, s, db->sync, ev), "kernel launch");
  HIP_TRY(hipEventRecord(db->done, s), "hipEventRecord");
  db->searched = true;
  return HMM_OK;
}

int hmm_search_group(const hmm_profile *const *p, hmm_db *const *db, const hmm_thresholds *t,
                     const hmm_results *out, int32_t n, hmm_stream stream) {
  if (n < 1) return fail(HMM_EINVAL, "n = %d; need at least one search", n);
  if (!p || !db || !t || !out) return fail(HMM_EINVAL, "NULL profile, db, thresholds or results array");
  // every check before any HIP call: a rejected group enqueues nothing
  for (int i = 0; i < n; i++) {
    if (!p[i] || !db[i]) return fail(HMM_EINVAL, "search %d: NULL profile or db", i);
    if (db[i]->data != db[0]->data) return fail(HMM_EINVAL, "search %d: handle of another database", i);
    for (int j = 0; j < i; j++)
      if (db[j] == db[i]) return fail(HMM_EINVAL, "searches %d and %d use the same handle", j, i);
    const hmm_thresholds &ti = t[i];
    if (std::isnan(ti.F1) || std::isnan(ti.F2) || std::isnan(ti.F3) || !(ti.F1 > 0) || !(ti.F2 > 0) ||
        !(ti.F3 > 0))
      return fail(HMM_EINVAL, "search %d: P-value cutoffs must be > 0", i);
    if (ti.bias_filter != 0 && ti.bias_filter != 1)
      return fail(HMM_EINVAL, "search %d: bias_filter = %d; need 0 or 1", i, ti.bias_filter);
    if (db[i]->n > 0 && (!out[i].msv || !out[i].vit || !out[i].fwd || !out[i].flags))
      return fail(HMM_EINVAL, "search %d: NULL output buffer", i);
    if (!int32_range_ok(p[i], db[i]))
      return fail(HMM_ERANGE, "search %d: longest target (%d) times largest emission score (%d) reaches 2^29", i,
                  db[i]->max_len, p[i]->s_max);
  }
  hipStream_t s = (hipStream_t)stream;
  if (db[0]->n == 0) return HMM_OK;
  std::vector<DevProfile> P(n);
  std::vector<DevDb> D(n);
  std::vector<DevOut> O(n);
  std::vector<const SearchSync *> Y(n);
  for (int i = 0; i < n; i++) {
    hmm_db *d = db[i];
    if (d->searched) HIP_TRY(hipStreamWaitEvent(s, d->done, 0), "hipStreamWaitEvent");
    if (d->lp_serial != p[i]->serial || d->lp_F[0] != t[i].F1 || d->lp_F[1] != t[i].F2 || d->lp_F[2] != t[i].F3) {
      if (d->searched) HIP_TRY(hipEventSynchronize(d->done), "hipEventSynchronize");
      for (int L = 0; L <= d->max_len; L++) length_params(p[i], &t[i], L < 1 ? 1 : L, &d->h_lp[L], nullptr);
      HIP_TRY(hipMemcpyAsync(d->d_lp, d->h_lp, sizeof(LenParams) * ((size_t)d->max_len + 1),
                             hipMemcpyHostToDevice, s),
              "hipMemcpyAsync(length table)");
      d->lp_serial = p[i]->serial;
      d->lp_F[0] = t[i].F1;
      d->lp_F[1] = t[i].F2;
      d->lp_F[2] = t[i].F3;
    }
    P[i] = p[i]->dev;
    D[i] = chunk_of(d->dev, 0, d->n, 0);
    O[i] = DevOut{out[i].msv,    out[i].vit,  out[i].fwd,        out[i].flags,
                  out[i].counts, out[i].bias, t[i].bias_filter, fuse_tail(d->fused_tail, t[i])};
    Y[i] = &d->sync;
  }
  HIP_TRY(launch_search_group(P.data(), D.data(), O.data(), n, s, Y.data()), "kernel launch");
  for (int i = 0; i < n; i++) {
    HIP_TRY(hipEventRecord(db[i]->done, s), "hipEventRecord");
    db[i]->searched = true;
  }
  return HMM_OK;
}

int hmm_count(const hmm_profile *p, hmm_db *db, const hmm_domain *dom, const int32_t *n_dom, int32_t max_dom,
              const int16_t *aln, uint32_t *counts, hmm_stream stream) {
  if (!p || !db || !dom || !n_dom || !aln || !counts) return fail(HMM_EINVAL, "NULL argument");
  if (max_dom < 0) return fail(HMM_EINVAL, "max_dom = %d", max_dom);
  hipStream_t s = (hipStream_t)stream;
  if (db->searched) HIP_TRY(hipStreamWaitEvent(s, db->done, 0), "hipStreamWaitEvent");
  if (max_dom > 0 && db->n > 0) HIP_TRY(launch_count(p->dev, db->dev, dom, n_dom, max_dom, aln, counts, s), "kernel launch");
  return HMM_OK;
}

int hmm_rebuild(const hmm_profile_desc *prior, const uint32_t *counts, double A, double B, double *match,
                double *insert, double *trans) {
  int rc = validate_desc(prior);
  if (rc) return rc;
  if (!counts || !match || (prior->M > 1 && (!insert || !trans))) return fail(HMM_EINVAL, "NULL argument");
  if (!(A > 0.0) || !(B > 0.0) || !std::isfinite(A) || !std::isfinite(B))
    return fail(HMM_EINVAL, "prior weights must be finite and > 0");
  const int M = prior->M;
  const uint32_t *cm = counts, *ci = counts + (size_t)M * kAlpha, *ct = ci + (size_t)(M - 1) * kAlpha;
  // e'(a) = (c(a) + w p(a)) / (sum c + w) over each row (or transition group)
  auto row = [](const uint32_t *c, const double *prev, int n, double w, double *out) {
    double tot = 0.0;
    for (int a = 0; a < n; a++) tot += (double)c[a];
    for (int a = 0; a < n; a++) out[a] = ((double)c[a] + w * prev[a]) / (tot + w);
  };
  for (int k = 0; k < M; k++) row(cm + (size_t)k * kAlpha, prior->match + (size_t)k * kAlpha, kAlpha, A,
                                  match + (size_t)k * kAlpha);
  for (int k = 0; k + 1 < M; k++) {
    row(ci + (size_t)k * kAlpha, prior->insert + (size_t)k * kAlpha, kAlpha, A, insert + (size_t)k * kAlpha);
    const uint32_t *c = ct + (size_t)k * 7;
    const double *t = prior->trans + (size_t)k * 7;
    double *o = trans + (size_t)k * 7;
    row(c, t, 3, B, o);           // MM MI MD
    row(c + 3, t + 3, 2, B, o + 3);   // IM II
    row(c + 5, t + 5, 2, B, o + 5);   // DM DD
  }
  return HMM_OK;
}

}  // extern "C"

namespace {

// Shared body of hmm_decode and hmm_decode_static.  With `fixed` set the
// wave slots live in the file-scope scratch array (kStaticDecodeBytes) and
// nothing is allocated; otherwise in the database's decode scratch, grown
// on demand.
int decode_impl(const hmm_profile *p, hmm_db *db, const uint8_t *flags, uint8_t mask, const hmm_decode_out *out,
                hmm_stream stream, bool fixed) {
  if (!p || !db || !out) return fail(HMM_EINVAL, "NULL profile, db or out");
  if (!out->dom || !out->n_dom) return fail(HMM_EINVAL, "NULL dom or n_dom");
  if (out->max_dom < 0) return fail(HMM_EINVAL, "max_dom = %d", out->max_dom);
  // one scratch slot per resident wave, four per workgroup
  const int64_t slot_dw = decode_slot_dw(p->dev.Q32, db->max_len);
  const size_t slot_bytes = (size_t)slot_dw * 4;
  const size_t budget = fixed ? kStaticDecodeBytes : kDecodeScratchMax;
  int64_t nslots = decode_max_waves(p->dev);
  nslots = std::min<int64_t>(nslots, (int64_t)(budget / slot_bytes));
  nslots = std::min<int64_t>(nslots, (db->n + 3) / 4 * 4);
  nslots = nslots / 4 * 4;
  if (db->n > 0 && nslots < 4) {
    if (fixed)
      return fail(HMM_ERANGE, "hmm_decode_static: 4 waves of %zu bytes (M = %d, longest target %d) exceed the "
                  "%zu-byte static scratch", slot_bytes, p->dev.M, db->max_len, kStaticDecodeBytes);
    return fail(HMM_ENOMEM, "decode scratch: %zu bytes per wave exceed the budget", slot_bytes);
  }
  float *base = nullptr;
  if (fixed && db->n > 0) HIP_TRY(static_decode_scratch(&base), "hipGetSymbolAddress(scratch)");
  hipStream_t s = (hipStream_t)stream;
  // serialise with the searches on this database (lists, counters, scratch)
  if (db->searched) HIP_TRY(hipStreamWaitEvent(s, db->done, 0), "hipStreamWaitEvent");
  DevDecode d{};
  d.dom = out->dom;
  d.max_dom = out->max_dom;
  d.n_dom = out->n_dom;
  d.exp_dom = out->exp_dom;
  d.pp = out->pp;
  d.aln = out->aln;
  d.sel_flags = flags;
  d.sel_mask = mask;
  d.rt1 = HMM_RT1;
  d.rt2 = HMM_RT2;
  if (db->n > 0) {
    // the loop and move probabilities of each length (profile-independent)
    if (db->lp_serial == 0) {
      if (db->searched) HIP_TRY(hipEventSynchronize(db->done), "hipEventSynchronize");
      const hmm_thresholds all{1.0, 1.0, 1.0, 0};
      for (int L = 0; L <= db->max_len; L++) length_params(p, &all, L < 1 ? 1 : L, &db->h_lp[L], nullptr);
      HIP_TRY(hipMemcpyAsync(db->d_lp, db->h_lp, sizeof(LenParams) * ((size_t)db->max_len + 1),
                             hipMemcpyHostToDevice, s),
              "hipMemcpyAsync(length table)");
      db->lp_serial = p->serial;
      db->lp_F[0] = db->lp_F[1] = db->lp_F[2] = 1.0;
    }
    if (!fixed) {
      const size_t need = (size_t)nslots * slot_bytes;
      if (need > db->dec_bytes) {
        if (db->searched) HIP_TRY(hipEventSynchronize(db->done), "hipEventSynchronize");
        if (db->dec_mem) HIP_TRY(hipFree(db->dec_mem), "hipFree(decode scratch)");
        db->dec_mem = nullptr;
        db->dec_bytes = 0;
        hipError_t e = hipMalloc(&db->dec_mem, need);
        if (e != hipSuccess)
          return e == hipErrorOutOfMemory ? fail(HMM_ENOMEM, "decode scratch of %zu bytes", need)
                                          : fail_hip(e, "hipMalloc(decode scratch)");
        db->dec_bytes = need;
      }
      base = (float *)db->dec_mem;
    }
    d.scratch = base;
    d.slot_dw = slot_dw;
    d.nslots = (int32_t)nslots;
  }
  HIP_TRY(launch_decode(p->dev, db->dev, d, s), "kernel launch");
  HIP_TRY(hipEventRecord(db->done, s), "hipEventRecord");
  db->searched = true;
  return HMM_OK;
}

}  // namespace

extern "C" {

int hmm_decode(const hmm_profile *p, hmm_db *db, const uint8_t *flags, uint8_t mask, const hmm_decode_out *out,
               hmm_stream stream) {
  return decode_impl(p, db, flags, mask, out, stream, false);
}

int hmm_decode_static(const hmm_profile *p, hmm_db *db, const uint8_t *flags, uint8_t mask,
                      const hmm_decode_out *out, hmm_stream stream) {
  return decode_impl(p, db, flags, mask, out, stream, true);
}

}  // extern "C"
