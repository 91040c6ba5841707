// HIP kernels (gfx950) of the profile-HMM search cascade and their launcher.
//
// One wavefront scores one target.  The model dimension (profile cells) is
// spread across the 64 lanes; database rows (residues) are processed in
// order.  Every wave-uniform quantity (target index, length, residue, the
// special states N/B/E/J/C) lives in scalar registers; branches on it are
// uniform.
//
//  MSV      the uint8 recurrence rewritten exactly in packed fp16 (small
//           integers), two cells per VGPR: one add and one 3-way maximum
//           per cell pair; each lane position follows one DP diagonal, so
//           no cross-lane move is needed (striped layout for large M).
//  Viterbi  packed saturating int16, two cells per VGPR; delete chain by
//           lazy propagation across slots.
//  Rescore  the Viterbi recurrence in int32 with a -2^30 floor.
//  Forward  fp32 probabilities with exact power-of-two rescaling; the
//           delete chain crosses slots through a DPP prefix scan of affine
//           maps, E through a DPP sum.
//
// Cell layout (see hmm_host.cpp): packed kernels use slot 2*lane+half and
// cell slot*Q + q (MSV's diagonal layout aside); 32-bit kernels use
// slot = lane and cell lane*Q + q.  The
// left neighbour of vector q is vector q-1 of the same slot, except q = 0,
// which takes vector Q-1 of the previous slot: one cross-lane shift per
// state per row.
#include <hip/hip_runtime.h>

#include <cmath>
#include <vector>

#include "hmm_device.h"
#include "hmm_internal.h"

namespace hmmgpu {
namespace {


// ============================================================================ MSV
//
// Per row i (residue a), with previous-row values v and xB (uint8 semantics,
// (+)/(-) saturating):
//   xBe = xB (-) ENTRY8;  v_k = (max(v_{k-1}, xBe) (+) BIAS8) (-) COST8_k(a)
//   xE = max v; overflow if xE >= 255 - BIAS8; xJ = max(xJ, xE (-) EXIT8);
//   xB = max(BASE8 (-) MOVE8, xJ (-) MOVE8)
//
// Exact reformulation in fp16 (every quantity is an integer of magnitude
// below 2048, so fp16 adds and maxima are exact).  Rows are only computed
// while every cell is below the overflow line 255 - BIAS8, so v_{k-1} (+)
// BIAS8 never saturates and only xBe can reach the 255 ceiling.  With
// E = BIAS8 - COST8 and Bx = min(xBe, 255 - BIAS8):
//   v_k = max(v_{k-1} + E, Bx + E, 0).
// The kernel keeps w = v - Bx, so that
//   w_k = max3(w_{k-1} + E, E, -Bx)
// is one packed add and one packed 3-way maximum (v_pk_maximum3_f16) per
// pair of cells, with E read straight from the table.  A running maximum of
// all cells (one more 3-way maximum per two vectors) is compared each row
// against the smallest value that could change xB or overflow; only then is
// the wave-wide maximum taken, xB updated and w re-based to the new Bx.
// A predecessor value w = 0 (v = Bx) or w = -Bx (v = 0) both give cell 0 its
// correct value max(E, -Bx), so cell 0 needs no special case, and padding
// cells (E = -1024) stay at w = -Bx, below every real cell.
//
// Two layouts of the cells over the 64 lanes x 2 halves x Q vectors:
//  DIAG (M + 1 <= 128 Q): MSV cells depend only on their diagonal
//    predecessor, so each of the P = 128 Q positions follows one diagonal of
//    the DP matrix: at row r position p holds cell (p + r) mod P, and its
//    predecessor is the same position's previous value.  No cross-lane
//    operation is needed.  The table row of residue a holds
//    D[c] = (E_c, E_{(c + P/2) mod P}) for c in [0, P); position dword
//    k = q*64 + lane (halves: diagonals k and k + P/2) reads D[k + r mod P/2],
//    and every P/2 rows the two halves of each state dword swap roles.  The
//    padding cell between cell M-1 and cell 0 (P >= M + 1) keeps diagonals
//    apart.
//  striped (larger M): slot 2*lane + half holds cells slot*Q + q; vector 0
//    takes vector Q-1 of the previous slot through one DPP lane shift and
//    one v_alignbit per row.
typedef _Float16 h16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ h16x2 as_h2(uint32_t v) { return __builtin_bit_cast(h16x2, v); }
__device__ __forceinline__ uint32_t as_u(h16x2 v) { return __builtin_bit_cast(uint32_t, v); }
__device__ __forceinline__ h16x2 h2_splat(int v) {
  const _Float16 h = (_Float16)(float)v;
  return h16x2{h, h};
}
__device__ __forceinline__ h16x2 h2_max3(h16x2 a, h16x2 b, h16x2 c) {
  return __builtin_elementwise_maximum(__builtin_elementwise_maximum(a, b), c);
}
__device__ __forceinline__ int h2_hmax(h16x2 v) { return (int)(float)__builtin_elementwise_maximum(v.x, v.y); }

// Composition-bias score of one target (nats; result in every lane): the
// forward probability ratio of a two-state null model (background, or the
// profile's mean match composition with odds r(a) = P.bias_r[a]; start
// 63/64 : 1/64, switch 1/64 per residue) against the background,
//   beta = ln (pi G_0 G_1 ... G_{L-1} 1),  G_0 = diag(1, r(x_0)),
//   G_i = [[63/64, r(x_i)/64], [1/64, 63/64 r(x_i)]].
// Each lane multiplies the 2x2 matrices of one contiguous segment of the
// target, then the segments are multiplied in order by a tree over the
// lanes; products are kept in [2^-20, 2^20] by exact power-of-two scaling
// with the exponents summed.
constexpr float kS8f = (float)(3.0 / M_LN2);

struct Mat2 {
  float a, b, c, d;   // [[a, b], [c, d]]
  int e;              // the product is this matrix times 2^e
};

__device__ __forceinline__ void mat2_mul(Mat2 &p, float ga, float gb, float gc, float gd, int ge) {
  const float a = fmaf(p.a, ga, p.b * gc), b = fmaf(p.a, gb, p.b * gd);
  const float c = fmaf(p.c, ga, p.d * gc), d = fmaf(p.c, gb, p.d * gd);
  p.a = a;
  p.b = b;
  p.c = c;
  p.d = d;
  p.e += ge;
  const float mx = fmaxf(fmaxf(a, b), fmaxf(c, d));
  if (mx > 0x1p20f || mx < 0x1p-20f) {
    int ex;
    (void)frexpf(mx, &ex);
    if (mx == 0.0f) ex = 0;
    const float s = ldexpf(1.0f, -ex);
    p.a *= s;
    p.b *= s;
    p.c *= s;
    p.d *= s;
    p.e += ex;
  }
}

__device__ float bias_score(const DevProfile &P, const uint8_t *x, int L, int lane) {
  constexpr float w = 1.0f / 64.0f, st = 63.0f / 64.0f;
  const int seg = (L + kWave - 1) / kWave;
  const int i0 = lane * seg, i1 = min(L, i0 + seg);
  Mat2 m{1.0f, 0.0f, 0.0f, 1.0f, 0};
  for (int i = i0; i < i1; i++) {   // lane-divergent, no cross-lane operation inside
    const float r = P.bias_r[x[i]];
    if (i == 0)
      mat2_mul(m, 1.0f, 0.0f, 0.0f, r, 0);
    else
      mat2_mul(m, st, w * r, w, st * r, 0);
  }
  for (int dd = 1; dd < kWave; dd <<= 1) {
    const float qa = __shfl_down(m.a, dd), qb = __shfl_down(m.b, dd), qc = __shfl_down(m.c, dd);
    const float qd = __shfl_down(m.d, dd);
    const int qe = __shfl_down(m.e, dd);
    if ((lane & (2 * dd - 1)) == 0 && lane + dd < kWave) mat2_mul(m, qa, qb, qc, qd, qe);
  }
  const float s0 = fmaf(st, m.a, w * m.c), s1 = fmaf(st, m.b, w * m.d);
  const float beta = logf(s0 + s1) + (float)m.e * (float)M_LN2;
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, beta), 0));
}

// ---------------------------------------------------------------- MSV table reads
// The diagonal layout's table rows are read with ds_read_addtid_b32, whose
// address is M0 + offset + 4 * lane: the wave-uniform part (residue row and
// diagonal offset) goes into M0 with one scalar move, so a row's reads cost
// no vector instruction.  The compiler does not see these loads in its
// wait-count tracking, so they are confined to straight-line code: the
// reads of row r+1 are issued before row r's arithmetic and waited for
// (s_waitcnt lgkmcnt(0)) right after it, before any branch.  No read is in
// flight at a branch, a merge or a loop edge, so no copy or reuse of a
// register can race with a read into it.  M0 is otherwise only written by
// the compiler right before its own uses (lane writes of the atomic-add
// scan), never carried across this code.
// A scalar write of M0 needs one wait state before an add-TID LDS
// instruction reads it (the s_nop).
template <int K, int Q>
__device__ __forceinline__ void lds_load_tid(uint32_t (&c)[Q], int base, int ofs) {
  asm volatile("s_add_u32 m0, %0, %1\n\ts_nop 0" ::"s"(base), "s"(ofs));
#pragma unroll
  for (int q = 0; q < Q; q++) asm volatile("ds_read_addtid_b32 %0 offset:%1" : "=v"(c[q]) : "i"(q * kWave * 4 + K));
}
// compile-time row offset, passed to the table-read functor
template <int K>
struct RowK {
  static constexpr int v = K;
};

// Lane j: dword j + 1 of the residue stream (lane 63: the next chunk's first
// dword), so the four rows of dword j find their successor's residue with one
// read and no branch at the chunk's end.
__device__ __forceinline__ uint32_t next_dwords(uint32_t cur, uint32_t nxt) {
  const int first = __builtin_amdgcn_readlane((int)nxt, 0);
  return (uint32_t)__builtin_amdgcn_update_dpp(first, (int)cur, 0x130 /* wave_shl:1 */, 0xf, 0xf, false);
}
template <int Q>
__device__ __forceinline__ void lds_wait(uint32_t (&c)[Q]) {
  asm volatile("s_waitcnt lgkmcnt(0)" ::);
#pragma unroll
  for (int q = 0; q < Q; q++) asm volatile("" : "+v"(c[q]));
}

// Row driver of the diagonal MSV: residues four to a dword as in drive_rows,
// table buffers in alternation, the rows of a dword taken in pairs.
// load(RowK<K>{}, buf, a) reads residue a's table entries for the row K rows
// after the current position; step(n) advances the position by n rows.
// row(cur, next, kind) computes a row from `cur`, waits for the reads into
// `next` (issued just before), then tests: kind 0 = first row of a pair (no
// test), 1 = second row of a pair (tests both), 2 = a row on its own (start
// or end of a run; tested).  Returns true if a row stopped the driver
// (`stop` = the last row computed) or the limit (a multiple of 4) was
// reached (`stop` = limit - 1).  The residue chunks are loaded two ahead,
// so the successor dwords of a chunk are at hand without waiting.  A chunk
// that holds none of the target's rows is not fetched: its load re-reads a
// chunk already in the cache and no row uses the value, so reads run at
// most 255 bytes past a target, inside the database's 1 KB zero tail.
// Plain (cached) loads: the lines a target shares with its neighbours in
// the length-sorted database, which neighbouring waves of the same block
// score at about the same time, are then fetched from HBM once.
template <int Q, typename Load, typename Step, typename Row>
__device__ __forceinline__ bool drive_pairs(const uint8_t *x, int L, int r0, int limit, int &stop, int lane,
                                            uint32_t (&ba)[Q], uint32_t (&bb)[Q], Load load, Step step, Row row) {
  auto code = [](uint32_t w, int r) { return (int)((w >> (8 * r)) & 0xffu); };
  int r = r0;
  for (; (r & 3) != 0; r++) {
    if (r >= L) return false;
    load(RowK<0>{}, ba, uni((int)x[r]));
    step(1);
    lds_wait(ba);
    if (row(ba, ba, 2)) {
      stop = r;
      return true;
    }
  }
  if (r >= L) return false;
  const int cs = r & ~255;
  const uint32_t *p = (const uint32_t *)(x + cs);
  // chunk k of the target from cs (its residues cs + 256 k ...), or chunk
  // `own` when chunk k holds no row
  auto chunk = [&](int k, int own) { return p[(size_t)(cs + 256 * k < L ? k : own) * kWave + lane]; };
  uint32_t cur = chunk(0, 0);
  uint32_t nxt = chunk(1, 0);
  uint32_t nn = chunk(2, 0);
  uint32_t sh = next_dwords(cur, nxt);
  int j0 = (r & 255) >> 2;
  uint32_t w = (uint32_t)__builtin_amdgcn_readlane((int)cur, j0);
  load(RowK<0>{}, ba, code(w, 0));
  lds_wait(ba);
  for (int c0 = cs;; c0 += 256) {
    const int nfull = min(kWave, (L - c0) >> 2);      // whole dwords of rows in this chunk
    const int jlim = min(nfull, (limit - c0) >> 2);   // ... before the limit
    for (int j = j0; j < jlim; j++) {
      const uint32_t wn = (uint32_t)__builtin_amdgcn_readlane((int)sh, j);
      load(RowK<1>{}, bb, code(w, 1));
      row(ba, bb, 0);
      load(RowK<2>{}, ba, code(w, 2));
      if (__builtin_expect(row(bb, ba, 1), 0)) {
        stop = c0 + 4 * j + 1;
        return true;
      }
      load(RowK<3>{}, bb, code(w, 3));
      row(ba, bb, 0);
      load(RowK<4>{}, ba, code(wn, 0));
      if (__builtin_expect(row(bb, ba, 1), 0)) {
        stop = c0 + 4 * j + 3;
        return true;
      }
      step(4);
      w = wn;
    }
    if (jlim < nfull) {
      stop = c0 + 4 * jlim - 1;
      return true;
    }
    if (nfull < kWave) {  // the target's last 0..3 rows (row 0's table already in ba)
      const int rt = c0 + 4 * nfull;
      if (rt >= L) return false;
      if (rt >= limit) {
        stop = rt - 1;
        return true;
      }
      for (int k = 0; rt + k < L; k++) {
        if (k) {
          load(RowK<0>{}, ba, code(w, k));
          lds_wait(ba);
        }
        step(1);
        if (row(ba, ba, 2)) {
          stop = rt + k;
          return true;
        }
      }
      return false;
    }
    if (c0 + 256 >= L) return false;
    j0 = 0;
    cur = nxt;
    nxt = nn;
    nn = chunk(((c0 - cs) >> 8) + 3, ((c0 - cs) >> 8) + 1);
    sh = next_dwords(cur, nxt);
  }
}

// Runs of consecutive (sorted) targets for the MSV waves, taken from the
// launch's work counter, so that waves slowed by other kernels on their CU,
// or by longer targets, take fewer.  A run is 8 targets, or fewer where the
// waves would otherwise get fewer than 4 runs each.  When there are no more
// runs than waves (a small database), wave w takes run w and no counter is
// used: the atomics alone would outlast the work (5,000 targets at M = 77:
// 0.23 against 0.13 ms).  Measured and not kept: a first run by wave index
// before the counter's (C2 MSV 1.51 against 1.30 ms), and a plain read of
// the counter before each bump, to leave without an atomic once the runs
// are gone (1.65 ms).
constexpr int kMsvRun = 8;
struct MsvRuns {
  int32_t *work;
  int n, run, nw, nruns;
  __device__ MsvRuns(int32_t *w, int n_) : work(w), n(n_) {
    nw = uni((int)gridDim.x * (int)(blockDim.x >> 6));
    run = max(1, min(kMsvRun, n / (4 * nw)));
    nruns = (n + run - 1) / run;
  }
  __device__ int first() const { return nruns <= nw ? wave_id() : wave_fetch_add(work, 1); }
  __device__ int next() const { return nruns <= nw ? nruns : wave_fetch_add(work, 1); }
};

struct MsvResult {
  int raw;
  bool ovf;
};

// Diagonal-layout MSV of one target, in two passes.
//
// Fast pass: every row with the entry value of the first row and no test
// at all; at the end, one test of the running maximum against the first
// trigger value T (the smallest cell value that could change xB or
// overflow).  If no cell reached T, xB never changed and no cell came near
// the overflow line, so the pass is exactly the recurrence and its maximum
// gives the score.  Background targets reach T with probability ~2^-19
// (about 19 bits above the score distribution's location); homologs and
// other high scorers do, and take the exact pass from the start.  Cells
// past T may lose fp16 exactness or saturate to +inf in the fast pass:
// rounding is monotone, so the maximum still compares at or above T.
//
// Exact pass: rows come in pairs and the trigger test runs once per pair,
// on two running maxima (even rows, odd rows).  When a pair fires and its
// first row already reached the trigger, the second row was computed with
// the old Bx; since xB only grows and
//   v'_k = max(v_{k-1} + E, Bx' + E, 0) = max(v_k, Bx' + E)   (Bx' >= Bx),
// that row is corrected in place from its own table entries: in units of
// the new Bx, w' = max(w + Bx - Bx', E).  Then the second row is tested
// again against the new trigger value.
template <int Q>
__device__ __forceinline__ MsvResult msv_target_diag(const DevProfile &P, const uint8_t *x, int L, const LenParams &lp,
                                                     int lane, uint32_t (&ca)[Q], uint32_t (&cb)[Q]) {
  constexpr int kHalf = Q * kWave;   // P/2: dwords per half table row
  constexpr int kRowB = 2 * kHalf * 4;  // bytes per residue in the table
  const int entry8 = P.entry8, exit8 = P.exit8;
  const int ovf_line = 255 - P.bias8;
  auto splat = [](int v) -> uint32_t { return (uint32_t)uni((int)as_u(h2_splat(v))); };
  const int mv = lp.move8;
  const int base = max(kBase8 - mv, 0);
  int xJt = 0;
  int Bx = min(max(base - entry8, 0), max(ovf_line, 0));
  bool ovf = ovf_line <= 0;
  h16x2 acc_e = as_h2(splat(-Bx)), acc_o = acc_e;
  if (!ovf) {
    h16x2 w[Q];
#pragma unroll
    for (int q = 0; q < Q; q++) w[q] = acc_e;
    uint32_t nbx = splat(-Bx);
    auto trigger_thr = [&]() { return splat(min(ovf_line, max(xJt, kBase8) + 4) - Bx - 1); };
    uint32_t thr = trigger_thr();
    // xJ from the largest cell m so far, and the Bx it gives the next row
    auto settle = [&](int m) {
      xJt = max(xJt, max(m - exit8, 0));
      return min(max(max(base, max(xJt - mv, 0)) - entry8, 0), ovf_line);
    };
    // running maximum: a tree of 3-way maxima where Q allows (depth 2 at
    // Q = 6 instead of a chain of 3), the same instruction count
    auto fold = [&](h16x2 &acc) {
      if constexpr (Q % 3 == 0) {
        h16x2 p[Q / 3];
#pragma unroll
        for (int j = 0; j < Q / 3; j++) p[j] = h2_max3(w[3 * j], w[3 * j + 1], w[3 * j + 2]);
#pragma unroll
        for (int j = 0; j + 1 < Q / 3; j += 2) acc = h2_max3(acc, p[j], p[j + 1]);
        if ((Q / 3) & 1) acc = __builtin_elementwise_maximum(acc, p[Q / 3 - 1]);
      } else {
#pragma unroll
        for (int q = 0; q + 1 < Q; q += 2) acc = h2_max3(acc, w[q], w[q + 1]);
        if (Q & 1) acc = __builtin_elementwise_maximum(acc, w[Q - 1]);
      }
    };
    auto fired = [&]() { return any_lane(as_u(h2_max3(acc_o, as_h2(thr), acc_e)) != thr); };
    // byte offset of the next load's row inside the residue's table row:
    // 4 (row mod P/2); the driver stops at every multiple of P/2 rows, so at
    // most one (discarded) read lies one dword row past P/2, still inside
    // the residue's table row of P dwords
    int lofs = 0;
    // Empty asm statements that "modify" the row state order the code: the
    // next row's reads are issued before this row's arithmetic, and the wait
    // for them comes after it, so the read latency hides behind the row.
    auto pin = [&]() {
#pragma unroll
      for (int q = 0; q < Q; q++) asm volatile("" : "+v"(w[q]));
    };
    auto load = [&](auto k, uint32_t(&c)[Q], int a) {
      lds_load_tid<4 * decltype(k)::v>(c, a * kRowB, uni(lofs));
      pin();
    };
    auto step = [&](int n) { lofs = uni(lofs + 4 * n); };   // kept uniform: an SGPR
    // the rows' arithmetic: every add, then every maximum, so that no
    // maximum waits on the add just before it (a dependent packed op needs
    // a wait state on gfx950)
    auto advance = [&](const uint32_t(&c)[Q]) {
      h16x2 t[Q];
#pragma unroll
      for (int q = 0; q < Q; q++) t[q] = w[q] + as_h2(c[q]);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int q = 0; q < Q; q++) w[q] = h2_max3(t[q], as_h2(c[q]), as_h2(nbx));
    };
    // at the end of every phase of P/2 rows the halves of each state dword
    // swap diagonals
    auto next_phase = [&](int stop) -> int {
      const int r = stop + 1;
      lofs = 4 * (r % kHalf);
      if (lofs == 0) {
#pragma unroll
        for (int q = 0; q < Q; q++) {
          const uint32_t u = as_u(w[q]);
          w[q] = as_h2(__builtin_amdgcn_alignbit(u, u, 16));
        }
      }
      return r;
    };
    // ---- fast pass
    bool exact = false;
    {
      auto frow = [&](const uint32_t(&c)[Q], uint32_t(&next)[Q], int) -> bool {
        advance(c);
        fold(acc_e);
        pin();
        lds_wait(next);
        return false;
      };
      int r = 0;
      for (;;) {
        int stop = 0;
        const int limit = (r / kHalf + 1) * kHalf;
        if (!drive_pairs(x, L, r, limit, stop, lane, ca, cb, load, step, frow)) break;
        r = next_phase(stop);
        if (r >= L) break;
      }
      exact = any_lane(as_u(__builtin_elementwise_maximum(acc_e, as_h2(thr))) != thr);
    }
    // ---- exact pass, from the first row again
    if (__builtin_expect(exact, 0)) {
#pragma unroll
      for (int q = 0; q < Q; q++) w[q] = as_h2(nbx);
      acc_e = acc_o = as_h2(nbx);
      lofs = 0;
    }
    auto row = [&](const uint32_t(&c)[Q], uint32_t(&next)[Q], int kind) -> bool {
      advance(c);
      fold(kind == 1 ? acc_o : acc_e);
      pin();
      lds_wait(next);
      if (__builtin_expect(kind == 0 || !fired(), 1)) return false;
      if (kind == 2 || !any_lane(as_u(__builtin_elementwise_maximum(acc_e, as_h2(thr))) != thr)) return true;
      // the pair's first row reached the trigger: settle it, correct the second row
      const int m = wave_max_i32(h2_hmax(acc_e)) + Bx;
      if (m >= ovf_line) {
        ovf = true;
        return true;
      }
      const int nBx = settle(m);
      if (nBx != Bx) {
        const h16x2 d = as_h2(splat(Bx - nBx));
#pragma unroll
        for (int q = 0; q < Q; q++) w[q] = __builtin_elementwise_maximum(w[q] + d, as_h2(c[q]));
        acc_e += d;
        acc_o += d;
        fold(acc_o);
        Bx = nBx;
        nbx = splat(-Bx);
      }
      thr = trigger_thr();
      return fired();
    };
    for (int r = 0; exact;) {
      int stop = 0;
      const int limit = (r / kHalf + 1) * kHalf;   // end of the current phase
      if (!drive_pairs(x, L, r, limit, stop, lane, ca, cb, load, step, row)) break;
      if (ovf) break;
      const int m = wave_max_i32(h2_hmax(__builtin_elementwise_maximum(acc_e, acc_o))) + Bx;
      if (m >= ovf_line) {
        ovf = true;
        break;
      }
      const int nBx = settle(m);
      if (nBx != Bx) {  // re-base w and the running maxima to the new Bx
        const h16x2 d = as_h2(splat(Bx - nBx));
#pragma unroll
        for (int q = 0; q < Q; q++) w[q] += d;
        acc_e += d;
        acc_o += d;
        Bx = nBx;
        nbx = splat(-Bx);
      }
      thr = trigger_thr();
      r = next_phase(stop);
      if (r >= L) break;
    }
  }
  MsvResult res{255, ovf};
  if (!ovf) {
    const int m = wave_max_i32(h2_hmax(__builtin_elementwise_maximum(acc_e, acc_o))) + Bx;
    const int xJ = max(m - exit8, 0);
    res.raw = max(xJ - mv, 0);
  }
  return res;
}

template <int Q, bool DIAG>
__global__ void __launch_bounds__(1024) msv_kernel(DevProfile P, DevDb db, DevOut out) {
  constexpr int kHalf = Q * kWave;                 // P/2 in DIAG, dwords per table row otherwise
  constexpr int kRow = DIAG ? 2 * kHalf : kHalf;   // dwords per residue in the table
  extern __shared__ uint32_t lds[];
  {
    const uint4 *src = (const uint4 *)P.msv;
    uint4 *dst = (uint4 *)lds;
    for (int i = threadIdx.x; i < kAlpha * kRow / 4; i += blockDim.x) dst[i] = src[i];
  }
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int entry8 = P.entry8, exit8 = P.exit8;
  const int ovf_line = 255 - P.bias8;
  const uint32_t *tab = lds + lane;
  const int n = (int)db.n;
  // table buffers of the diagonal path (kept defined: its driver's exits use them)
  uint32_t da[Q], dbuf[Q];
#pragma unroll
  for (int q = 0; q < Q; q++) da[q] = dbuf[q] = 0;
  // packed fp16 pair (v, v) as a wave-uniform dword
  auto splat = [](int v) -> uint32_t { return (uint32_t)uni((int)as_u(h2_splat(v))); };
  // Targets in runs (MsvRuns).  The next target's length and start are read
  // during the current target's epilogue, so a target starts with one round
  // trip (its length parameters and first residue chunks, in parallel)
  // instead of three.
  const MsvRuns runs(&db.counters[CNT_WORK_MSV], n);
  int t = runs.first() * runs.run;
  int tend = min(t + runs.run, n);
  int Lnext = 0;
  int64_t snext = 0;
  if (t < n) {
    Lnext = uni(db.len[t]);
    snext = db.start[t];
  }
  while (t < n) {
    const int L = Lnext;
    const uint8_t *x = db.res + snext;
    const LenParams lp = db.lp[L];
    MsvResult res;
    if constexpr (DIAG) {
      res = msv_target_diag<Q>(P, x, L, lp, lane, da, dbuf);
    } else {  // striped layout
      const int mv = lp.move8;
      const int base = max(kBase8 - mv, 0);
      int xJt = 0;
      int Bx = min(max(base - entry8, 0), max(ovf_line, 0));
      bool ovf = ovf_line <= 0;
      h16x2 acc = as_h2(splat(-Bx));
      if (!ovf) {
        h16x2 w[Q];
#pragma unroll
        for (int q = 0; q < Q; q++) w[q] = acc;
        uint32_t nbx = splat(-Bx);
        // Trigger: some cell reaches T, the smallest value that could change
        // xB or overflow; in w units, some w > T - Bx - 1.
        auto trigger_thr = [&]() { return splat(min(ovf_line, max(xJt, kBase8) + 4) - Bx - 1); };
        uint32_t thr = trigger_thr();
        auto load = [&](uint32_t(&c)[Q], int a) {
          const uint32_t *row = (const uint32_t *)((const char *)tab + a * (kRow * 4));
#pragma unroll
          for (int q = 0; q < Q; q++) c[q] = row[q * kWave];
        };
        auto advance = [&](const uint32_t(&c)[Q]) {
          const uint32_t sh = slot_up16(as_u(w[Q - 1]));
#pragma unroll
          for (int q = Q - 1; q >= 0; q--) {
            const h16x2 e = as_h2(c[q]);
            w[q] = h2_max3((q ? w[q - 1] : as_h2(sh)) + e, e, as_h2(nbx));
          }
#pragma unroll
          for (int q = 0; q + 1 < Q; q += 2) acc = h2_max3(acc, w[q], w[q + 1]);
          if (Q & 1) acc = __builtin_elementwise_maximum(acc, w[Q - 1]);
        };
        auto fired = [&]() { return any_lane(as_u(__builtin_elementwise_maximum(acc, as_h2(thr))) != thr); };
        uint32_t ca[Q], cb[Q];
        // Fast pass, as in the diagonal layout: no test until the end; if
        // no cell reached the first trigger value, the pass is exact.
        {
          auto frow = [&](const uint32_t(&c)[Q]) -> bool {
            advance(c);
            return false;
          };
          int stop = 0;
          (void)drive_rows(x, L, 0, 0, stop, lane, ca, cb, load, frow);
        }
        const bool exact = fired();
        if (__builtin_expect(exact, 0)) {   // exact pass from the first row again
#pragma unroll
          for (int q = 0; q < Q; q++) w[q] = as_h2(nbx);
          acc = as_h2(nbx);
        }
        // One row of the exact pass.  Only w and the running maximum change
        // here, on every row: a trigger stops the row driver; the caller then
        // updates xJ and xB, re-bases w, and resumes at the next row.
        auto row = [&](const uint32_t(&c)[Q]) -> bool {
          advance(c);
          return __builtin_expect(fired(), 0);
        };
        int r = 0;
        for (; exact;) {
          int stop = 0;
          if (!drive_rows(x, L, r, 0, stop, lane, ca, cb, load, row)) break;
          const int m = wave_max_i32(h2_hmax(acc)) + Bx;      // largest cell so far
          if (m >= ovf_line) {
            ovf = true;
            break;
          }
          xJt = max(xJt, max(m - exit8, 0));
          const int nBx = min(max(max(base, max(xJt - mv, 0)) - entry8, 0), ovf_line);
          if (nBx != Bx) {  // re-base w (and the running maximum) to the new Bx
            const h16x2 d = as_h2(splat(Bx - nBx));
#pragma unroll
            for (int q = 0; q < Q; q++) w[q] += d;
            acc += d;
            Bx = nBx;
            nbx = splat(-Bx);
          }
          thr = trigger_thr();
          r = stop + 1;
          if (r >= L) break;
        }
      }
      res.ovf = ovf;
      res.raw = 255;
      if (!ovf) {
        const int m = wave_max_i32(h2_hmax(acc)) + Bx;
        const int xJ = max(m - exit8, 0);
        res.raw = max(xJ - mv, 0);
      }
    }
    const bool ovf = res.ovf;
    const int raw = res.raw;
    int tn = t + 1;
    if (tn >= tend) {
      tn = runs.next() * runs.run;
      tend = min(tn + runs.run, n);
    }
    if (tn < n) {
      Lnext = uni(db.len[tn]);
      snext = db.start[tn];
    }
    const bool pass = ovf || raw >= lp.thr8;
    const uint8_t fl = (pass ? HMM_MSV_PASS : 0) | (ovf ? HMM_MSV_OVF : 0);
    // sorted order: neighbouring waves score neighbouring targets, so these
    // stores fill whole cache lines; results_kernel writes the caller's order
    db.flags_sorted[t] = fl;
    db.msv_sorted[t] = (int16_t)raw;
    // with the composition-bias filter on, MSV passes go to the filter's
    // list (the overflow list, unused until Viterbi) instead of Viterbi's
    if (pass) {
      const bool bf = out.bias_filter != 0;
      (bf ? db.list_ovf : db.list_vit)[wave_fetch_add(&db.counters[bf ? CNT_OVF : CNT_VIT], 1)] = t;
    }
    t = tn;
  }
}

// ---------------------------------------------------------------- MSV of a group of profiles
// Several searches of one database by different profiles of the same
// diagonal instance (Q): one wave scores a target against G profiles at
// once.  The residue stream, its scalar handling and M0 are shared: the
// tables sit interleaved in LDS as [residue][profile][P], so one M0 serves
// the G profiles' reads (profile g at immediate offset g * P * 4).  Each
// profile keeps its own state, running maxima, xJ/xB and trigger value,
// exactly as msv_target_diag, and its own outputs and survivor list.  A
// profile that overflows stops taking part in the tests (its trigger value
// becomes +inf); its cells keep being computed and are ignored.
template <int G>
struct MsvGroup {
  DevProfile P[G];
  DevDb db[G];
  DevOut out[G];
};

template <int K, int Q, int G>
__device__ __forceinline__ void lds_load_group(uint32_t (&c)[G * Q], int base, int ofs) {
  asm volatile("s_add_u32 m0, %0, %1\n\ts_nop 0" ::"s"(base), "s"(ofs));
#pragma unroll
  for (int g = 0; g < G; g++)
#pragma unroll
    for (int q = 0; q < Q; q++)
      asm volatile("ds_read_addtid_b32 %0 offset:%1" : "=v"(c[g * Q + q]) : "i"((g * 2 * Q + q) * kWave * 4 + K));
}

// Eight waves per SIMD (two blocks per CU), as the single-profile kernel:
// the G profiles' scalar state would otherwise take more than the 100 SGPRs
// that allows, and leave one block per CU.
template <int Q, int G>
__global__ void __launch_bounds__(1024) __attribute__((amdgpu_waves_per_eu(8, 8)))
msv_group_kernel(MsvGroup<G> A) {
  constexpr int kHalf = Q * kWave;       // P/2
  constexpr int kRowB = 2 * kHalf * 4;   // bytes per residue and profile
  extern __shared__ uint32_t lds[];
  for (int g = 0; g < G; g++) {
    const uint32_t *src = A.P[g].msv;
    for (int i = threadIdx.x; i < kAlpha * 2 * kHalf; i += blockDim.x) {
      const int a = i / (2 * kHalf), c = i - a * (2 * kHalf);
      lds[(a * G + g) * (2 * kHalf) + c] = src[i];
    }
  }
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const DevDb &D0 = A.db[0];
  const int n = (int)D0.n;
  auto splat = [](int v) -> uint32_t { return (uint32_t)uni((int)as_u(h2_splat(v))); };
  constexpr uint32_t kInf2 = 0x7c007c00u;   // (+inf, +inf): never fires
  uint32_t ca[G * Q], cb[G * Q];
#pragma unroll
  for (int i = 0; i < G * Q; i++) ca[i] = cb[i] = 0;
  // targets in runs, as in the single-profile kernel (the work counter is
  // the first profile's)
  const MsvRuns runs(&D0.counters[CNT_WORK_MSV], n);
  int t = runs.first() * runs.run;
  int tend = min(t + runs.run, n);
  int Lnext = 0;
  int64_t snext = 0;
  if (t < n) {
    Lnext = uni(D0.len[t]);
    snext = D0.start[t];
  }
  while (t < n) {
    const int L = Lnext;
    const uint8_t *x = D0.res + snext;
    int mv[G], base[G], xJt[G], Bx[G], ovf_line[G];
    bool ovf[G];
    uint32_t nbx[G], thr[G];
    h16x2 w[G][Q], acc_e[G], acc_o[G];
    auto trigger_thr = [&](int g) {
      return ovf[g] ? kInf2 : splat(min(ovf_line[g], max(xJt[g], kBase8) + 4) - Bx[g] - 1);
    };
#pragma unroll
    for (int g = 0; g < G; g++) {
      mv[g] = A.db[g].lp[L].move8;
      base[g] = max(kBase8 - mv[g], 0);
      ovf_line[g] = 255 - A.P[g].bias8;
      xJt[g] = 0;
      Bx[g] = min(max(base[g] - A.P[g].entry8, 0), max(ovf_line[g], 0));
      ovf[g] = ovf_line[g] <= 0;
      acc_e[g] = acc_o[g] = as_h2(splat(-Bx[g]));
#pragma unroll
      for (int q = 0; q < Q; q++) w[g][q] = acc_e[g];
      nbx[g] = splat(-Bx[g]);
      thr[g] = trigger_thr(g);
    }
    auto settle = [&](int g, int m) {
      xJt[g] = max(xJt[g], max(m - A.P[g].exit8, 0));
      return min(max(max(base[g], max(xJt[g] - mv[g], 0)) - A.P[g].entry8, 0), ovf_line[g]);
    };
    auto fold = [&](h16x2 &acc, const h16x2 (&v)[Q]) {
#pragma unroll
      for (int q = 0; q + 1 < Q; q += 2) acc = h2_max3(acc, v[q], v[q + 1]);
      if (Q & 1) acc = __builtin_elementwise_maximum(acc, v[Q - 1]);
    };
    auto fired = [&](int g) { return any_lane(as_u(h2_max3(acc_o[g], as_h2(thr[g]), acc_e[g])) != thr[g]); };
    auto rebase = [&](int g, int nBx) {
      const h16x2 d = as_h2(splat(Bx[g] - nBx));
#pragma unroll
      for (int q = 0; q < Q; q++) w[g][q] += d;
      acc_e[g] += d;
      acc_o[g] += d;
      Bx[g] = nBx;
      nbx[g] = splat(-nBx);
    };
    int lofs = 0;
    auto pin = [&]() {
#pragma unroll
      for (int g = 0; g < G; g++)
#pragma unroll
        for (int q = 0; q < Q; q++) asm volatile("" : "+v"(w[g][q]));
    };
    auto load = [&](auto k, uint32_t(&c)[G * Q], int a) {
      lds_load_group<4 * decltype(k)::v, Q, G>(c, a * (G * kRowB), uni(lofs));
      pin();
    };
    auto step = [&](int n) { lofs = uni(lofs + 4 * n); };   // kept uniform: an SGPR
    // every add, then every maximum (as in the single-profile kernel)
    auto advance = [&](const uint32_t(&c)[G * Q]) {
      h16x2 tt[G][Q];
#pragma unroll
      for (int g = 0; g < G; g++)
#pragma unroll
        for (int q = 0; q < Q; q++) tt[g][q] = w[g][q] + as_h2(c[g * Q + q]);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int g = 0; g < G; g++)
#pragma unroll
        for (int q = 0; q < Q; q++) w[g][q] = h2_max3(tt[g][q], as_h2(c[g * Q + q]), as_h2(nbx[g]));
    };
    auto next_phase = [&](int stop) -> int {
      const int r = stop + 1;
      lofs = 4 * (r % kHalf);
      if (lofs == 0) {  // the halves of every state dword swap diagonals
#pragma unroll
        for (int g = 0; g < G; g++)
#pragma unroll
          for (int q = 0; q < Q; q++) {
            const uint32_t u = as_u(w[g][q]);
            w[g][q] = as_h2(__builtin_amdgcn_alignbit(u, u, 16));
          }
      }
      return r;
    };
    bool all_ovf0 = true;
#pragma unroll
    for (int g = 0; g < G; g++) all_ovf0 = all_ovf0 && ovf[g];
    // Fast pass (as in msv_target_diag): every profile without tests; if
    // none reached its first trigger value, the pass is exact for all.
    bool exact = false;
    if (!all_ovf0) {
      auto frow = [&](const uint32_t(&c)[G * Q], uint32_t(&next)[G * Q], int) -> bool {
        advance(c);
#pragma unroll
        for (int g = 0; g < G; g++) fold(acc_e[g], w[g]);
        pin();
        lds_wait(next);
        return false;
      };
      for (int r = 0;;) {
        int stop = 0;
        const int limit = (r / kHalf + 1) * kHalf;
        if (!drive_pairs(x, L, r, limit, stop, lane, ca, cb, load, step, frow)) break;
        r = next_phase(stop);
        if (r >= L) break;
      }
      uint64_t any = 0;
#pragma unroll
      for (int g = 0; g < G; g++)
        any |= __builtin_amdgcn_ballot_w64(as_u(__builtin_elementwise_maximum(acc_e[g], as_h2(thr[g]))) != thr[g]);
      exact = any != 0;
    }
    if (__builtin_expect(exact, 0)) {   // exact pass for every profile, from the first row again
#pragma unroll
      for (int g = 0; g < G; g++) {
#pragma unroll
        for (int q = 0; q < Q; q++) w[g][q] = as_h2(nbx[g]);
        acc_e[g] = acc_o[g] = as_h2(nbx[g]);
      }
      lofs = 0;
    }
    auto row = [&](const uint32_t(&c)[G * Q], uint32_t(&next)[G * Q], int kind) -> bool {
      advance(c);
#pragma unroll
      for (int g = 0; g < G; g++) fold(kind == 1 ? acc_o[g] : acc_e[g], w[g]);
      pin();
      lds_wait(next);
      if (kind == 0) return false;
      uint64_t any = 0;
#pragma unroll
      for (int g = 0; g < G; g++)
        any |= __builtin_amdgcn_ballot_w64(as_u(h2_max3(acc_o[g], as_h2(thr[g]), acc_e[g])) != thr[g]);
      if (__builtin_expect(!any, 1)) return false;
      bool stop = false;
#pragma unroll
      for (int g = 0; g < G; g++) {
        if (!fired(g)) continue;
        if (kind == 2 || !any_lane(as_u(__builtin_elementwise_maximum(acc_e[g], as_h2(thr[g]))) != thr[g])) {
          stop = true;   // the tested row reached the trigger: the caller settles it
          continue;
        }
        // the pair's first row reached the trigger: settle it, correct the second row
        const int m = wave_max_i32(h2_hmax(acc_e[g])) + Bx[g];
        if (m >= ovf_line[g]) {
          ovf[g] = true;
          thr[g] = kInf2;
          continue;
        }
        const int nBx = settle(g, m);
        if (nBx != Bx[g]) {
          const h16x2 d = as_h2(splat(Bx[g] - nBx));
#pragma unroll
          for (int q = 0; q < Q; q++) w[g][q] = __builtin_elementwise_maximum(w[g][q] + d, as_h2(c[g * Q + q]));
          acc_e[g] += d;
          acc_o[g] += d;
          fold(acc_o[g], w[g]);
          Bx[g] = nBx;
          nbx[g] = splat(-nBx);
        }
        thr[g] = trigger_thr(g);
        if (fired(g)) stop = true;
      }
      return stop;
    };
    for (int r = 0; exact;) {
      bool all_ovf = true;
#pragma unroll
      for (int g = 0; g < G; g++) all_ovf = all_ovf && ovf[g];
      if (all_ovf) break;
      int stop = 0;
      const int limit = (r / kHalf + 1) * kHalf;   // end of the current phase
      if (!drive_pairs(x, L, r, limit, stop, lane, ca, cb, load, step, row)) break;
#pragma unroll
      for (int g = 0; g < G; g++) {   // settle every profile whose trigger fired on the stop row
        if (!fired(g)) continue;
        const int m = wave_max_i32(h2_hmax(__builtin_elementwise_maximum(acc_e[g], acc_o[g]))) + Bx[g];
        if (m >= ovf_line[g]) {
          ovf[g] = true;
          thr[g] = kInf2;
          continue;
        }
        const int nBx = settle(g, m);
        if (nBx != Bx[g]) rebase(g, nBx);
        thr[g] = trigger_thr(g);
      }
      r = next_phase(stop);
      if (r >= L) break;
    }
    int tn = t + 1;
    if (tn >= tend) {
      tn = runs.next() * runs.run;
      tend = min(tn + runs.run, n);
    }
    if (tn < n) {
      Lnext = uni(D0.len[tn]);
      snext = D0.start[tn];
    }
#pragma unroll
    for (int g = 0; g < G; g++) {
      int raw = 255;
      if (!ovf[g]) {
        const int m = wave_max_i32(h2_hmax(__builtin_elementwise_maximum(acc_e[g], acc_o[g]))) + Bx[g];
        raw = max(max(m - A.P[g].exit8, 0) - mv[g], 0);
      }
      const DevDb &Dg = A.db[g];
      const DevOut &Og = A.out[g];
      const bool pass = ovf[g] || raw >= Dg.lp[L].thr8;
      const uint8_t fl = (pass ? HMM_MSV_PASS : 0) | (ovf[g] ? HMM_MSV_OVF : 0);
      Dg.flags_sorted[t] = fl;
      Dg.msv_sorted[t] = (int16_t)raw;
      if (pass) {
        const bool bf = Og.bias_filter != 0;
        (bf ? Dg.list_ovf : Dg.list_vit)[wave_fetch_add(&Dg.counters[bf ? CNT_OVF : CNT_VIT], 1)] = t;
      }
    }
    t = tn;
  }
}

// Composition-bias filter on the MSV passes (list_ovf, count CNT_OVF): the
// bias score of each, and the ones whose MSV score less the bias still
// reaches the cutoff (or that overflowed MSV) go on to Viterbi's list.
__global__ void __launch_bounds__(256) bias_kernel(DevProfile P, DevDb db, DevOut out) {
  const int lane = threadIdx.x & 63;
  const int count = uni(__atomic_load_n(&db.counters[CNT_OVF], __ATOMIC_RELAXED));
  for (;;) {
    const int idx = wave_fetch_add(&db.counters[CNT_WORK_OVF], 1);
    if (idx >= count) break;
    const int t = uni(db.list_ovf[idx]);
    const int L = uni(db.len[t]);
    const LenParams lp = db.lp[L];
    const float beta = bias_score(P, db.res + db.start[t], L, lane);
    uint8_t fl = (uint8_t)uni(db.flags_sorted[t]);
    const int raw = (int)uni((int)db.msv_sorted[t]);
    const bool go = (fl & HMM_MSV_OVF) || (float)raw - kS8f * fmaxf(beta, 0.0f) >= (float)lp.thr8;
    if (go) fl |= HMM_BIAS_PASS;
    db.flags_sorted[t] = fl;
    if (out.bias) out.bias[uni(db.perm[t])] = beta;
    if (go) db.list_vit[wave_fetch_add(&db.counters[CNT_VIT], 1)] = t;
  }
}

// The overflow list and its counters start empty for Viterbi.
__global__ void reset_ovf(int32_t *c) {
  if (threadIdx.x == 0) {
    c[CNT_OVF] = 0;
    c[CNT_WORK_OVF] = 0;
  }
}

// ============================================================================ Viterbi int16
//
// Per row, with previous-row M, I, D and xB, every add saturating on its own:
//   M_k = sat(max(sat(xB+ENTRY16), sat(M_{k-1}+MM), sat(I_{k-1}+IM), sat(D_{k-1}+DM)) + msc_k(a))
//   I_k = sat(max(sat(M_k+MI), sat(I_k+II)) + isc_k(a))
//   D_k = max(sat(M_{k-1}+MD), sat(D_{k-1}+DD))          (current row)
//   xE = max_k M_k (delete transitions are <= 0, so D_k <= max M);
//   xJ = max(xJ, sat(xE+EJ16)); xB = max(sat(MOVE16), sat(xJ+MOVE16))
// overflow if some M or I reaches 32767.  xB depends on max(xJ, 0) only,
// so the wave-wide maximum is taken only when a cell reaches the value that
// would raise it.  The delete chain is computed inside each slot, then
// propagated across slots until no lane changes (exact: sat is monotone).
//
// Delete floor: D only feeds match cells (through D->M) and later deletes
// (through D->D <= 0), and every match cell of this and every later row
// includes the entry value xBe, which never decreases.  So a delete value
// d <= tau = xBe - max_k DM_k, and everything the chain derives from it, can
// never change a match cell: the kernel keeps D' = max(D, tau) instead of D
// (the floored recurrence's fixed point is exactly max(D, tau), since
// sat(tau + DD) <= tau), and sat(D' + DM) differs from sat(D + DM) only
// where both are <= xBe.  M, I, xE and the overflow test are unchanged, and
// the lazy propagation stops as soon as the chains that cross a slot
// boundary fall to the floor, instead of running every chain to its end.

// Threads per block of the Viterbi kernel.  Large instances run one wave per
// SIMD (4 waves per block): each wave may then use the whole register file,
// architectural and accumulation registers, and spills go to accumulation
// registers rather than to scratch memory.
template <int Q>
constexpr int kThreads16 = Q >= 16 ? 256 : 512;
// Instances whose transition planes, all but D->D, are read from LDS every
// row instead of being held in registers (D->D, which the lazy delete
// propagation also reads, stays in registers): 120 fewer registers at 20
// vectors per lane, so that two waves share a SIMD and hide each other's
// waits.
template <int Q>
constexpr bool kTrLds16 = Q == 16 || Q == 20;
template <int Q>
constexpr int kMinWaves16 = kTrLds16<Q> ? 2 : 1;
// Threads per block of the one-wave rescore and Forward kernels.
constexpr int kThreads32 = 512;

struct VitResult {
  int raw;
  bool ovf;
};


template <int Q, bool TRL = false>
__device__ __forceinline__ VitResult vit16_target(const uint32_t *__restrict__ emit, const uint32_t (&tr)[TR_N][Q],
                                                  const DevProfile &P, const uint8_t *x, int L,
                                                  const LenParams &lp, int lane, const uint32_t *ltr = nullptr) {
  uint32_t M[Q], I[Q], D[Q];
#pragma unroll
  for (int q = 0; q < Q; q++) M[q] = I[q] = D[q] = kNegNeg;
  uint32_t accM = kNegNeg, accI = kNegNeg;
  const int mv = lp.move16, ej = P.ej16, entry = P.entry16;
  int xJt = kNeg16;
  int xB = sat16(mv);
  uint32_t xbe2 = splat16(sat16(xB + entry));
  auto floor_of = [&](int xbe) { return splat16(min(xbe - P.dm_max16, 32767)); };
  uint32_t tau2 = floor_of(sat16(xB + entry));
  int T = min(-ej + 1, 32767);
  uint32_t tm1 = splat16(T - 1);
  bool ovf = false;
  auto load = [&](uint32_t(&e)[2 * Q], int a) {
    const uint32_t *er = emit + a * (2 * Q * kWave);
#pragma unroll
    for (int q = 0; q < 2 * Q; q++) e[q] = er[q * kWave];
  };
  auto row = [&](const uint32_t(&em)[2 * Q]) -> bool {
    // LDS planes: an offset the compiler cannot see through keeps their
    // reads inside the row (loop-invariant reads would be hoisted back
    // into registers)
    int off = 0;
    if (TRL) asm volatile("" : "+v"(off));
    auto trv = [&](int k, int q) -> uint32_t { return TRL ? ltr[off + (k * Q + q) * kWave] : tr[k][q]; };
    const uint32_t msh = slot_up16(M[Q - 1]);
    const uint32_t ish = slot_up16(I[Q - 1]);
    const uint32_t dsh = slot_up16(D[Q - 1]);
#pragma unroll
    for (int q = Q - 1; q >= 0; q--) {
      const uint32_t pm = q ? M[q - 1] : msh, pi = q ? I[q - 1] : ish, pd = q ? D[q - 1] : dsh;
      uint32_t m = i16_max(xbe2, i16_adds(pm, trv(TR_MMIN, q)));
      m = i16_max(m, i16_adds(pi, trv(TR_IMIN, q)));
      m = i16_max(m, i16_adds(pd, trv(TR_DMIN, q)));
      const uint32_t mn = i16_adds(m, em[q]);
      const uint32_t in =
          i16_adds(i16_max(i16_adds(M[q], trv(TR_MI, q)), i16_adds(I[q], trv(TR_II, q))), em[Q + q]);
      accM = i16_max(accM, mn);
      accI = i16_max(accI, in);
      M[q] = mn;
      I[q] = in;
    }
    uint32_t dc = kNegNeg;
    const uint32_t din = slot_up16(M[Q - 1]);
    // the floor joins the M->D term, which does not depend on the chain:
    // the chain itself is one add and one maximum per vector
#pragma unroll
    for (int q = 0; q < Q; q++) {
      const uint32_t md = i16_max(i16_adds(q ? M[q - 1] : din, trv(TR_MDIN, q)), tau2);
      D[q] = i16_max(md, i16_adds(dc, tr[TR_DDIN][q]));
      dc = D[q];
    }
    // A chain can cross into the next slot only from a slot whose last
    // delete value is above the floor (sat(tau + DD) <= tau <= D): when every
    // slot's last value is at the floor, nothing is left to propagate.
    // (A test of whether some slot's first cell would improve, in front of
    // the loop, measured slower: C3 Viterbi 2.90-2.94 against 2.85-2.87 ms.)
    if (any_lane(D[Q - 1] != tau2)) {
      for (int it = 0; it < 2 * kWave; it++) {
        dc = slot_up16(D[Q - 1]);
        bool moved = true;
#pragma unroll
        for (int q = 0; q < Q; q++) {
          if (moved) {
            const uint32_t nd = i16_max(D[q], i16_adds(dc, tr[TR_DDIN][q]));
            moved = any_lane(nd != D[q]);
            D[q] = nd;
            dc = nd;
          }
        }
        if (!moved) break;
      }
    }
    if (__builtin_expect(any_lane(i16_max(accM, tm1) != tm1), 0)) {
      const int m = wave_max_i32(hmax16(accM));
      if (m >= 32767) return true;
      xJt = max(xJt, sat16(m + ej));
      xB = max(sat16(mv), sat16(xJt + mv));
      xbe2 = splat16(sat16(xB + entry));
      tau2 = floor_of(sat16(xB + entry));
      T = min(max(xJt, 0) - ej + 1, 32767);
      tm1 = splat16(T - 1);
    }
    return false;
  };
  uint32_t ea[2 * Q], eb[2 * Q];
  int stop;
  ovf = drive_rows(x, L, 0, 0, stop, lane, ea, eb, load, row);
  if (!ovf) ovf = any_lane(hmax16(accI) >= 32767);
  VitResult res;
  res.ovf = ovf;
  if (ovf) {
    res.raw = 32767;
  } else {
    const int m = wave_max_i32(hmax16(accM));
    res.raw = sat16(sat16(m + ej) + mv);
  }
  return res;
}

template <int Q, bool EMIT_LDS>
__global__ void __launch_bounds__(kThreads16<Q>, kMinWaves16<Q>) vit16_kernel(DevProfile P, DevDb db, DevOut out) {
  extern __shared__ uint32_t lds[];
  constexpr bool TRL = kTrLds16<Q>;
  static_assert(!(TRL && EMIT_LDS), "one LDS table per instance");
  const int lane = threadIdx.x & 63;
  // a launch with no target returns before staging its table
  const int count = uni(__atomic_load_n(&db.counters[CNT_VIT], __ATOMIC_RELAXED));
  if (count == 0) return;
  if (EMIT_LDS || TRL) {
    const uint4 *src = (const uint4 *)(EMIT_LDS ? P.vit_emit : P.vit_tr);
    const int n4 = (EMIT_LDS ? kAlpha * 2 : TR_N) * Q * kWave / 4;
    uint4 *dst = (uint4 *)lds;
    for (int i = threadIdx.x; i < n4; i += blockDim.x) dst[i] = src[i];
    __syncthreads();
  }
  const uint32_t *emit = (EMIT_LDS ? (const uint32_t *)lds : P.vit_emit) + lane;
  uint32_t tr[TR_N][Q];
#pragma unroll
  for (int k = 0; k < TR_N; k++)
#pragma unroll
    for (int q = 0; q < Q; q++)
      tr[k][q] = (!TRL || k == TR_DDIN) ? P.vit_tr[(k * Q + q) * kWave + lane] : 0u;
  for (;;) {
    const int idx = wave_fetch_add(&db.counters[CNT_WORK_VIT], 1);
    if (idx >= count) break;
    const int t = uni(db.list_vit[idx]);
    const int L = uni(db.len[t]);
    if (db.prio_by_len) length_priority(L, db.max_len);
    const LenParams lp = db.lp[L];
    const VitResult r = vit16_target<Q, TRL>(emit, tr, P, db.res + db.start[t], L, lp, lane, (const uint32_t *)lds + lane);
    const bool pass = r.ovf || r.raw >= lp.thr16;
    const uint8_t fl =
        (uint8_t)(uni(db.flags_sorted[t]) | HMM_VIT_RAN | (pass ? HMM_VIT_PASS : 0) | (r.ovf ? HMM_VIT_OVF : 0));
    db.flags_sorted[t] = fl;
    out.vit[uni(db.perm[t])] = r.raw;
    if (r.ovf) db.list_ovf[wave_fetch_add(&db.counters[CNT_OVF], 1)] = t;
    if (pass) db.list_fwd[wave_fetch_add(&db.counters[CNT_FWD], 1)] = t;
  }
}

// ============================================================================ Viterbi int32 rescore
//
// The int16 recurrence in int32 with every add floored at -2^30 and no upper
// clamp; run on the targets that overflowed int16.  One wave per target, for
// profiles up to 12 vectors per lane (longer ones: hmm_coop.hip): emission
// rows come from LDS, prefetched a row ahead; transitions stay in registers.

__device__ __forceinline__ int fl32(int v) { return max(v, kNeg32); }

// One target's int32 Viterbi score (raw, before the null model), emission
// rows from `emit` (lane's column of [20][2][Q][64]), transitions `tr`.
template <int Q>
__device__ __forceinline__ int vit32_target(const int *emit, const int (&tr)[TR_N][Q], const DevProfile &P,
                                            const uint8_t *x, int L, const LenParams &lp, int lane) {
  auto TR = [&](int k, int q) -> int { return tr[k][q]; };
  const int mv = lp.move16, ej = P.ej16, entry = P.entry16;
  int M[Q], I[Q], D[Q];
#pragma unroll
  for (int q = 0; q < Q; q++) M[q] = I[q] = D[q] = kNeg32;
  int accM = kNeg32;
  int xJt = kNeg32;
  int xB = fl32(mv);
  int xbe = fl32(xB + entry);
  int tau = xbe - P.dm_max32;   // delete floor (as in the int16 kernel); >= xbe >= -2^30
  int T = -ej + 1;
  auto load = [&](int(&e)[2 * Q], int a) {
    const int *er = emit + a * (2 * Q * kWave);
#pragma unroll
    for (int q = 0; q < 2 * Q; q++) e[q] = er[q * kWave];
  };
  auto row = [&](const int(&em)[2 * Q]) -> bool {
    const int msh = lane_up_i(M[Q - 1]);
    const int ish = lane_up_i(I[Q - 1]);
    const int dsh = lane_up_i(D[Q - 1]);
    // The oracle floors every add at -2^30.  Here every add saturates
    // (v_add_i32 clamp), so no sum wraps, and only two floors remain: the
    // insert maximum's -2^30 and the delete floor tau.  A value below
    // -2^30 (after an impossible emission or transition) reaches only
    // maxima that hold a term >= -2^30 -- the match maximum includes xBe,
    // the insert maximum -2^30, the delete maximum tau -- so it is dropped
    // there exactly as the oracle's floored -2^30 is, and every state
    // that is not below -2^30 equals the oracle's.
#pragma unroll
    for (int q = Q - 1; q >= 0; q--) {
      const int pm = q ? M[q - 1] : msh, pi = q ? I[q - 1] : ish, pd = q ? D[q - 1] : dsh;
      const int m = max(max(xbe, sadd32(pm, TR(TR_MMIN, q))),
                        max(sadd32(pi, TR(TR_IMIN, q)), sadd32(pd, TR(TR_DMIN, q))));
      const int mn = sadd32(m, em[q]);
      const int in = sadd32(max(max(sadd32(M[q], TR(TR_MI, q)), sadd32(I[q], TR(TR_II, q))), kNeg32), em[Q + q]);
      accM = max(accM, mn);
      M[q] = mn;
      I[q] = in;
    }
    int dc = kNeg32;
    const int din = lane_up_i(M[Q - 1]);
#pragma unroll
    for (int q = 0; q < Q; q++) {
      D[q] = max(max(sadd32(q ? M[q - 1] : din, TR(TR_MDIN, q)), sadd32(dc, TR(TR_DDIN, q))), tau);
      dc = D[q];
    }
    // Chains crossing into the next lane: nothing moves unless some lane's
    // first cell improves, which this one test rules out in the common case.
    if (any_lane(lane_up_i(D[Q - 1]) + TR(TR_DDIN, 0) > D[0])) {
      for (int it = 0; it < kWave; it++) {
        dc = lane_up_i(D[Q - 1]);
        bool moved = true;
#pragma unroll
        for (int q = 0; q < Q; q++) {
          if (moved) {
            const int nd = max(D[q], dc + TR(TR_DDIN, q));   // D[q] >= tau >= -2^30 already
            moved = any_lane(nd != D[q]);
            D[q] = nd;
            dc = nd;
          }
        }
        if (!moved) break;
      }
    }
    if (any_lane(accM >= T)) {
      const int m = wave_max_i32(accM);
      xJt = max(xJt, fl32(m + ej));
      xB = max(fl32(mv), fl32(xJt + mv));
      xbe = fl32(xB + entry);
      tau = xbe - P.dm_max32;
      T = max(xJt, 0) - ej + 1;
    }
    return false;
  };
  int ea[2 * Q], eb[2 * Q];
  int stop;
  (void)drive_rows(x, L, 0, 0, stop, lane, ea, eb, load, row);
  const int m = wave_max_i32(accM);
  return fl32(fl32(m + ej) + mv);
}

template <int Q>
__device__ __forceinline__ void load_tr32(const DevProfile &P, int lane, int (&tr)[TR_N][Q]) {
#pragma unroll
  for (int k = 0; k < TR_N; k++)
#pragma unroll
    for (int q = 0; q < Q; q++) tr[k][q] = P.v32_tr[(k * Q + q) * kWave + lane];
}

template <int Q>
__global__ void __launch_bounds__(kThreads32) vit32_kernel(DevProfile P, DevDb db, DevOut out) {
  extern __shared__ int32_t lds32[];
  const int lane = threadIdx.x & 63;
  constexpr int kEmit = kAlpha * 2 * Q * kWave;   // dwords
  // a launch with no target (no int16 overflow) returns before staging its table
  const int count = uni(__atomic_load_n(&db.counters[CNT_OVF], __ATOMIC_RELAXED));
  if (count == 0) return;
  for (int i = threadIdx.x; i < kEmit / 4; i += blockDim.x) ((int4 *)lds32)[i] = ((const int4 *)P.v32_emit)[i];
  __syncthreads();
  const int *emit = (const int *)lds32 + lane;
  int tr[TR_N][Q];
  load_tr32<Q>(P, lane, tr);
  for (;;) {
    const int idx = wave_fetch_add(&db.counters[CNT_WORK_OVF], 1);
    if (idx >= count) break;
    const int t = uni(db.list_ovf[idx]);
    const int L = uni(db.len[t]);
    if (db.prio_by_len) length_priority(L, db.max_len);
    const LenParams lp = db.lp[L];
    out.vit[uni(db.perm[t])] = vit32_target<Q>(emit, tr, P, db.res + db.start[t], L, lp, lane);
  }
}

// ============================================================================ Forward fp32
//
// Probability space, 1 = the start state.  Per row (residue a):
//   M_k = e_k(a)/f(a) * (M_{k-1} MM + I_{k-1} IM + D_{k-1} DM + B entry)    (previous row)
//   I_k = i_k(a)/f(a) * (M_k MI + I_k II)                                    (previous row)
//   D_k = M_{k-1} MD + D_{k-1} DD                                            (current row)
//   E = sum_k (M_k + D_k); J = J loop + E/2; C = C loop + E/2; N = N loop;
//   B = (N + J) move.
// The delete chain runs inside each slot with a zero entry value; the values
// entering the slots follow from an inclusive scan of the affine maps
// x -> D_out + P x across lanes (P = product of the slot's DD), whose P part
// is profile-constant and precomputed.  Values are rescaled by an exact power
// of two whenever the largest special value leaves [2^-40, 2^40]; the removed
// exponents are summed.  Result: ln(C move) + (sum of exponents) ln 2, nats.

// Per-profile register state of the one-wave Forward: transitions, exit
// weights and the P part of the delete-chain scan (the lane's P before each
// of the six steps).
template <int Q>
struct FwdRegs {
  float tr[TR_N + 1][Q], gx[Q], pstep[6];
};

template <int Q>
__device__ __forceinline__ void load_fwd_regs(const DevProfile &P, int lane, FwdRegs<Q> &R) {
  const float *trp = P.f_tr + lane;
#pragma unroll
  for (int k = 0; k <= TR_N; k++)
#pragma unroll
    for (int q = 0; q < Q; q++) R.tr[k][q] = trp[(k * Q + q) * kWave];
#pragma unroll
  for (int q = 0; q < Q; q++) R.gx[q] = trp[(TR_EXIT * Q + q) * kWave];   // exit weights: E = sum M g
  float p = P.f_tr[(TR_N * Q + Q - 1) * kWave + lane];
#define HMM_PSTEP(I, CTRL, MASK) \
  R.pstep[I] = p;                \
  p = p * dpp_f<CTRL, MASK>(p, 1.0f);
  HMM_PSTEP(0, kRowShr1, 0xf)
  HMM_PSTEP(1, kRowShr2, 0xf)
  HMM_PSTEP(2, kRowShr4, 0xf)
  HMM_PSTEP(3, kRowShr8, 0xf)
  HMM_PSTEP(4, kRowBcast15, 0xa)
  HMM_PSTEP(5, kRowBcast31, 0xc)
#undef HMM_PSTEP
}

// One target's Forward score in nats (before the null model), emission
// rows from `emit` (lane's column of [20][2][Q][64]).
template <int Q>
__device__ __forceinline__ float fwd_target(const float *emit, const FwdRegs<Q> &R, const DevProfile &P,
                                            const uint8_t *x, int L, const LenParams &lp, int lane) {
  auto TR = [&](int k, int q) -> float { return R.tr[k][q]; };
  const float(&gx)[Q] = R.gx;
  const float(&pstep)[6] = R.pstep;
  const float entry_p = P.entry_p;
  const float loop = lp.loop_p, move = lp.move_p;
  float M[Q], I[Q], D[Q];
#pragma unroll
  for (int q = 0; q < Q; q++) M[q] = I[q] = D[q] = 0.0f;
  float N = 1.0f, B = move, J = 0.0f, C = 0.0f;
  int shift = 0;
  auto load = [&](float(&e)[2 * Q], int a) {
    const float *er = emit + a * (2 * Q * kWave);
#pragma unroll
    for (int q = 0; q < 2 * Q; q++) e[q] = er[q * kWave];
  };
  auto row = [&](const float(&em)[2 * Q]) -> bool {
    const float bent = B * entry_p;
    // the first cell's predecessors are the previous lane's last cells
    // (none in lane 0), read through the lane shift of each multiply-add
    float sm0 = bent;
    fmac_up3(sm0, D[Q - 1], TR(TR_DMIN, 0), I[Q - 1], TR(TR_IMIN, 0), M[Q - 1], TR(TR_MMIN, 0));
    float part = 0.0f;   // this lane's part of E: sum of M g (deletes included through g)
#pragma unroll
    for (int q = Q - 1; q >= 0; q--) {
      const float sm =
          q ? fmaf(M[q - 1], TR(TR_MMIN, q), fmaf(I[q - 1], TR(TR_IMIN, q), fmaf(D[q - 1], TR(TR_DMIN, q), bent)))
            : sm0;
      const float si = fmaf(M[q], TR(TR_MI, q), I[q] * TR(TR_II, q));
      M[q] = em[q] * sm;
      I[q] = em[Q + q] * si;
      part = fmaf(M[q], gx[q], part);
    }
    // delete chain inside the lane from a zero entry (the first cell's M
    // predecessor is the previous lane's new last M)
    D[0] = mul_up(M[Q - 1], TR(TR_MDIN, 0));
#pragma unroll
    for (int q = 1; q < Q; q++) D[q] = fmaf(M[q - 1], TR(TR_MDIN, q), D[q - 1] * TR(TR_DDIN, q));
    const float carry = lane_up_f(affine_scan_fused(D[Q - 1], pstep));
#pragma unroll
    for (int q = 0; q < Q; q++) D[q] = fmaf(carry, TR(TR_N, q), D[q]);
    const float E = wave_sum_fused(part);
    J = fmaf(J, loop, 0.5f * E);
    C = fmaf(C, loop, 0.5f * E);
    N = N * loop;
    B = (N + J) * move;
    const float big = fmaxf(fmaxf(fmaxf(E, J), fmaxf(C, N)), B);
    if (big > 0x1p40f || big < 0x1p-40f) {
      int ex;
      (void)frexpf(big, &ex);
      ex = uni(ex);
      const float s = ldexpf(1.0f, -ex);
#pragma unroll
      for (int q = 0; q < Q; q++) {
        M[q] *= s;
        I[q] *= s;
        D[q] *= s;
      }
      J *= s;
      C *= s;
      N *= s;
      B *= s;
      shift += ex;
    }
    return false;
  };
  float ea[2 * Q], eb[2 * Q];
  int stop;
  (void)drive_rows(x, L, 0, 0, stop, lane, ea, eb, load, row);
  return (float)(log((double)C * (double)move) + (double)shift * M_LN2);
}

template <int Q>
__global__ void __launch_bounds__(kThreads32) fwd_kernel(DevProfile P, DevDb db, DevOut out) {
  extern __shared__ float ldsf[];
  const int lane = threadIdx.x & 63;
  constexpr int kEmit = kAlpha * 2 * Q * kWave;
  // a launch with no target returns before staging its table
  const int count = uni(__atomic_load_n(&db.counters[CNT_FWD], __ATOMIC_RELAXED));
  if (count == 0) return;
  for (int i = threadIdx.x; i < kEmit / 4; i += blockDim.x) ((float4 *)ldsf)[i] = ((const float4 *)P.f_emit)[i];
  __syncthreads();
  const float *emit = (const float *)ldsf + lane;
  FwdRegs<Q> R;
  load_fwd_regs<Q>(P, lane, R);
  for (;;) {
    const int idx = wave_fetch_add(&db.counters[CNT_WORK_FWD], 1);
    if (idx >= count) break;
    const int t = uni(db.list_fwd[idx]);
    const int L = uni(db.len[t]);
    if (db.prio_by_len) length_priority(L, db.max_len);
    const LenParams lp = db.lp[L];
    const float f = fwd_target<Q>(emit, R, P, db.res + db.start[t], L, lp, lane);
    const bool pass = f > lp.fthr;
    const uint8_t fl = (uint8_t)(uni(db.flags_sorted[t]) | HMM_FWD_RAN | (pass ? HMM_FWD_PASS : 0));
    db.flags_sorted[t] = fl;
    out.fwd[uni(db.perm[t])] = f;
    if (pass) (void)wave_fetch_add(&db.counters[CNT_FWD_PASS], 1);
  }
}

// ============================================================================ fused tail
//
// For profiles of up to 384 nodes (3 int16 vectors per lane) the three
// stages after MSV run as one kernel: a wave takes an MSV survivor, scores
// it with the int16 Viterbi, rescores it in int32 at once if it overflowed,
// and runs Forward on it at once if it passed.  The staged kernels each wait
// for the longest target of the stage before them; here a target's stages
// follow each other without waiting for any other target, and a launch ends
// when its last wave's chain of stages does.  The three emission tables sit
// in LDS side by side (10 KB per vector of each: the int16 Viterbi's per
// int16 vector, the rescore's and Forward's per 32-bit vector);
// transitions are read per target and stage, so that no stage's
// registers stay live through the others.  Results, flags and counts are
// the staged kernels' (the survivor lists between the stages are not
// written).
template <int Q8>
constexpr int kThreadsTail = Q8 <= 2 ? 1024 : 512;

template <int Q8, int Q32>
__global__ void __launch_bounds__(kThreadsTail<Q8>) tail_kernel(DevProfile P, DevDb db, DevOut out) {
  extern __shared__ uint32_t ldst[];
  const int lane = threadIdx.x & 63;
  constexpr int n16 = kAlpha * 2 * Q8 * kWave, n32 = kAlpha * 2 * Q32 * kWave;   // dwords
  // a launch with no target returns before staging its tables
  const int count = uni(__atomic_load_n(&db.counters[CNT_VIT], __ATOMIC_RELAXED));
  if (count == 0) return;
  for (int i = threadIdx.x; i < n16 / 4; i += blockDim.x) ((uint4 *)ldst)[i] = ((const uint4 *)P.vit_emit)[i];
  for (int i = threadIdx.x; i < n32 / 4; i += blockDim.x) {
    ((uint4 *)(ldst + n16))[i] = ((const uint4 *)P.v32_emit)[i];
    ((uint4 *)(ldst + n16 + n32))[i] = ((const uint4 *)P.f_emit)[i];
  }
  __syncthreads();
  const uint32_t *e16 = ldst + lane;
  const int *e32 = (const int *)ldst + n16 + lane;
  const float *ef = (const float *)ldst + n16 + n32 + lane;
  for (;;) {
    const int idx = wave_fetch_add(&db.counters[CNT_WORK_VIT], 1);
    if (idx >= count) break;
    const int t = uni(db.list_vit[idx]);
    const int L = uni(db.len[t]);
    if (db.prio_by_len) length_priority(L, db.max_len);
    const LenParams lp = db.lp[L];
    const uint8_t *x = db.res + db.start[t];
    // the transition reads' lane offset, opaque to the compiler: otherwise
    // it keeps every read's address live through the loop
    int ln = lane;
    asm volatile("" : "+v"(ln));
    VitResult r;
    {
      uint32_t tr[TR_N][Q8];
#pragma unroll
      for (int k = 0; k < TR_N; k++)
#pragma unroll
        for (int q = 0; q < Q8; q++) tr[k][q] = P.vit_tr[(k * Q8 + q) * kWave + ln];
      r = vit16_target<Q8>(e16, tr, P, x, L, lp, lane);
    }
    const bool pass = r.ovf || r.raw >= lp.thr16;
    int vit = r.raw;
    if (r.ovf) {
      (void)wave_fetch_add(&db.counters[CNT_OVF], 1);
      int tr[TR_N][Q32];
      load_tr32<Q32>(P, ln, tr);
      vit = vit32_target<Q32>(e32, tr, P, x, L, lp, lane);
    }
    const int c = uni(db.perm[t]);
    out.vit[c] = vit;
    uint8_t fl = (uint8_t)(uni(db.flags_sorted[t]) | HMM_VIT_RAN | (pass ? HMM_VIT_PASS : 0) |
                           (r.ovf ? HMM_VIT_OVF : 0));
    if (pass) {
      (void)wave_fetch_add(&db.counters[CNT_FWD], 1);
      FwdRegs<Q32> R;
      load_fwd_regs<Q32>(P, ln, R);
      const float f = fwd_target<Q32>(ef, R, P, x, L, lp, lane);
      const bool fpass = f > lp.fthr;
      fl |= (uint8_t)(HMM_FWD_RAN | (fpass ? HMM_FWD_PASS : 0));
      out.fwd[c] = f;
      if (fpass) (void)wave_fetch_add(&db.counters[CNT_FWD_PASS], 1);
    }
    db.flags_sorted[t] = fl;
  }
}

// ============================================================================ small kernels

__global__ void clear_counters(int32_t *c, int nblocks) {
  for (int i = threadIdx.x; i < nblocks * CNT_N; i += blockDim.x) c[i] = 0;
}

__global__ void export_counts(const int32_t *c, int nblocks, int64_t *counts) {
  if (threadIdx.x == 0) {
    int64_t v[4] = {0, 0, 0, 0};
    for (int k = 0; k < nblocks; k++) {
      const int32_t *b = c + k * CNT_N;
      v[0] += b[CNT_VIT];
      v[1] += b[CNT_OVF];
      v[2] += b[CNT_FWD];
      v[3] += b[CNT_FWD_PASS];
    }
    for (int i = 0; i < 4; i++) counts[i] = v[i];
  }
}

// Results in the caller's order, once every stage of a search is done: each
// thread takes one caller index c and its sorted index iperm[c]; the flags
// and MSV score come from the sorted arrays the stages wrote, and Viterbi
// and Forward scores, written in caller order by those stages for the
// targets they scored, get INT32_MIN and NaN where the stage did not run.
// Reads of iperm and writes of every output are contiguous.
__global__ void __launch_bounds__(256) results_kernel(DevDb db, DevOut out) {
  const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= db.n) return;
  const int t = db.iperm[c];
  const uint8_t fl = db.flags_sorted[t];
  out.flags[c] = fl;
  out.msv[c] = db.msv_sorted[t];
  if (!(fl & HMM_VIT_RAN)) out.vit[c] = INT32_MIN;
  if (!(fl & HMM_FWD_RAN)) out.fwd[c] = __builtin_nanf("");
}

// ============================================================================ launcher

int g_num_cu = 0;

int num_cu() {
  if (!g_num_cu) {
    int dev = 0;
    (void)hipGetDevice(&dev);
    (void)hipDeviceGetAttribute(&g_num_cu, hipDeviceAttributeMultiprocessorCount, dev);
    if (g_num_cu <= 0) g_num_cu = 256;
  }
  return g_num_cu;
}

template <typename K>
int blocks_per_cu(K kernel, int threads, size_t lds) {
  int nb = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, kernel, threads, lds) != hipSuccess || nb < 1) nb = 1;
  return nb;
}

template <int Q, bool DIAG>
hipError_t launch_msv(const DevProfile &P, const DevDb &db, const DevOut &o, hipStream_t s) {
  const int threads = 1024;
  const size_t lds = (size_t)kAlpha * Q * kWave * 4 * (DIAG ? 2 : 1);
  auto k = msv_kernel<Q, DIAG>;
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void *)k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  static int bpc = 0;
  if (!bpc) bpc = blocks_per_cu(k, threads, lds);
  int64_t blocks = (int64_t)bpc * num_cu();
  const int64_t cap = (db.n + threads / 64 - 1) / (threads / 64);
  if (blocks > cap) blocks = cap;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k, dim3((unsigned)blocks), dim3(threads), lds, s, P, db, o);
  return hipGetLastError();
}

template <int Q, int G>
hipError_t launch_msv_group_t(const DevProfile *P, const DevDb *db, const DevOut *o, hipStream_t s) {
  MsvGroup<G> A;
  for (int g = 0; g < G; g++) {
    A.P[g] = P[g];
    A.db[g] = db[g];
    A.out[g] = o[g];
  }
  const int threads = 1024;
  const size_t lds = (size_t)G * kAlpha * 2 * Q * kWave * 4;
  auto k = msv_group_kernel<Q, G>;
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void *)k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  static int bpc = 0;
  if (!bpc) bpc = blocks_per_cu(k, threads, lds);
  int64_t blocks = (int64_t)bpc * num_cu();
  const int64_t cap = (db[0].n + threads / 64 - 1) / (threads / 64);
  if (blocks > cap) blocks = cap;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k, dim3((unsigned)blocks), dim3(threads), lds, s, A);
  return hipGetLastError();
}

template <int Q>
hipError_t launch_vit16(const DevProfile &P, const DevDb &db, const DevOut &o, hipStream_t s) {
  constexpr bool kLds = Q <= 8;
  const int threads = kThreads16<Q>;
  const size_t lds = kLds ? (size_t)kAlpha * 2 * Q * kWave * 4 : kTrLds16<Q> ? (size_t)TR_N * Q * kWave * 4 : 0;
  auto k = vit16_kernel<Q, kLds>;
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void *)k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  static int bpc = 0;
  if (!bpc) bpc = blocks_per_cu(k, threads, lds);
  int64_t blocks = (int64_t)bpc * num_cu();
  const int64_t cap = (db.n + threads / 64 - 1) / (threads / 64);
  if (blocks > cap) blocks = cap;
  hipLaunchKernelGGL(k, dim3((unsigned)blocks), dim3(threads), lds, s, P, db, o);
  return hipGetLastError();
}

// Persistent launch of a list kernel: as many blocks as fit, at most one
// wave per database target.
template <typename K>
hipError_t launch_list_kernel(K k, int threads, int &bpc, size_t lds, const DevProfile &P, const DevDb &db,
                              const DevOut &o, hipStream_t s) {
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void *)k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  if (!bpc) bpc = blocks_per_cu(k, threads, lds);
  int64_t blocks = (int64_t)bpc * num_cu();
  const int64_t cap = (db.n + threads / 64 - 1) / (threads / 64);
  if (blocks > cap) blocks = cap;
  hipLaunchKernelGGL(k, dim3((unsigned)blocks), dim3(threads), lds, s, P, db, o);
  return hipGetLastError();
}

// One-wave 32-bit kernels: the emission table in LDS (at most 120 KB, for
// 12 vectors per lane), transitions in registers.
template <int Q>
hipError_t launch_vit32(const DevProfile &P, const DevDb &db, const DevOut &o, hipStream_t s) {
  static_assert(Q <= 12, "longer profiles take the cooperative kernels");
  const size_t lds = (size_t)kAlpha * 2 * Q * kWave * 4;
  static int bpc = 0;
  return launch_list_kernel(vit32_kernel<Q>, kThreads32, bpc, lds, P, db, o, s);
}

template <int Q>
hipError_t launch_fwd(const DevProfile &P, const DevDb &db, const DevOut &o, hipStream_t s) {
  static_assert(Q <= 12, "longer profiles take the cooperative kernels");
  const size_t lds = (size_t)kAlpha * 2 * Q * kWave * 4;
  static int bpc = 0;
  return launch_list_kernel(fwd_kernel<Q>, kThreads32, bpc, lds, P, db, o, s);
}

// Fused tail (profiles of up to 3 int16 vectors per lane): the three
// emission tables in LDS, as many blocks as fit, at most one wave per target.
template <int Q8, int Q32>
hipError_t launch_tail_fused(const DevProfile &P, const DevDb &db, const DevOut &o, hipStream_t s) {
  const size_t lds = (size_t)kAlpha * 2 * kWave * 4 * (Q8 + 2 * Q32);
  static int bpc = 0;
  return launch_list_kernel(tail_kernel<Q8, Q32>, kThreadsTail<Q8>, bpc, lds, P, db, o, s);
}

// The int16 / 32-bit vector counts with a fused-tail instance.
bool tail_fused_instance(const DevProfile &P) {
  return (P.Q8 == 1 && P.Q32 <= 2) || (P.Q8 == 2 && (P.Q32 == 3 || P.Q32 == 4)) ||
         (P.Q8 == 3 && (P.Q32 == 5 || P.Q32 == 6));
}

hipError_t dispatch_tail_fused(const DevProfile &P, const DevDb &db, const DevOut &o, hipStream_t s) {
#define HMM_TAIL(a, b) \
  if (P.Q8 == a && P.Q32 == b) return launch_tail_fused<a, b>(P, db, o, s);
  HMM_TAIL(1, 1) HMM_TAIL(1, 2) HMM_TAIL(2, 3) HMM_TAIL(2, 4) HMM_TAIL(3, 5) HMM_TAIL(3, 6)
#undef HMM_TAIL
  return hipErrorInvalidValue;
}

#define HMM_Q8_CASES(X) X(1) X(2) X(3) X(4) X(5) X(6) X(7) X(8) X(10) X(12) X(14) X(16) X(20) X(24)
// One-wave instances of the 32-bit kernels; 14 and more vectors per lane
// (14, 16, 20, 24, 28, 32, 40, 48) run the cooperative ones.
#define HMM_Q32_CASES(X) X(1) X(2) X(3) X(4) X(5) X(6) X(8) X(10) X(12)

// MSV instances: diagonal layout up to 14 vectors per lane (table 10 KB per
// vector in LDS), striped above.
#define HMM_MSV_DIAG_CASES(X) X(1) X(2) X(3) X(4) X(5) X(6) X(7) X(8) X(10) X(12) X(14)
#define HMM_MSV_STRIPED_CASES(X) X(14) X(16) X(20) X(24)

hipError_t launch_bias(const DevProfile &P, const DevDb &db, const DevOut &o, hipStream_t s) {
  static int bpc = 0;
  if (!bpc) bpc = blocks_per_cu(bias_kernel, 256, 0);
  int64_t blocks = (int64_t)bpc * num_cu();
  const int64_t cap = (db.n + 3) / 4;
  if (blocks > cap) blocks = cap;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(bias_kernel, dim3((unsigned)blocks), dim3(256), 0, s, P, db, o);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(reset_ovf, dim3(1), dim3(64), 0, s, db.counters);
  return hipGetLastError();
}

hipError_t dispatch_msv(const DevProfile &P, const DevDb &db, const DevOut &o, hipStream_t s) {
  if (P.msv_diag) {
    switch (P.Qm) {
#define HMM_CASE(q) \
  case q:           \
    return launch_msv<q, true>(P, db, o, s);
      HMM_MSV_DIAG_CASES(HMM_CASE)
#undef HMM_CASE
    }
  } else {
    switch (P.Qm) {
#define HMM_CASE(q) \
  case q:           \
    return launch_msv<q, false>(P, db, o, s);
      HMM_MSV_STRIPED_CASES(HMM_CASE)
#undef HMM_CASE
    }
  }
  return hipErrorInvalidValue;
}

// Largest group of profiles the group MSV kernel takes at Q vectors per lane
// (diagonal layout): as many tables as two 1024-thread blocks per CU can hold
// in LDS (about 60 KB each) within the 64 registers per lane of eight waves
// per SIMD, at most 4; 1 = no group instance.
int msv_group_max(int Q) { return Q == 1 ? 4 : Q == 2 ? 3 : Q == 3 ? 2 : 1; }

hipError_t dispatch_msv_group(const DevProfile *P, const DevDb *db, const DevOut *o, int G, hipStream_t s) {
  const int Q = P[0].Qm;
#define HMM_GROUP(q, g) \
  if (Q == q && G == g) return launch_msv_group_t<q, g>(P, db, o, s);
  HMM_GROUP(1, 2) HMM_GROUP(1, 3) HMM_GROUP(1, 4) HMM_GROUP(2, 2) HMM_GROUP(2, 3) HMM_GROUP(3, 2)
#undef HMM_GROUP
  return hipErrorInvalidValue;
}

hipError_t dispatch_vit16(const DevProfile &P, const DevDb &db, const DevOut &o, hipStream_t s) {
  switch (P.Q8) {
#define HMM_CASE(q) \
  case q:           \
    return launch_vit16<q>(P, db, o, s);
    HMM_Q8_CASES(HMM_CASE)
#undef HMM_CASE
  }
  return hipErrorInvalidValue;
}

hipError_t dispatch_vit32(const DevProfile &P, const DevDb &db, const DevOut &o, hipStream_t s) {
  if (coop_instance(P.Q32)) return launch_vit32_coop(P, db, o, s);
  switch (P.Q32) {
#define HMM_CASE(q) \
  case q:           \
    return launch_vit32<q>(P, db, o, s);
    HMM_Q32_CASES(HMM_CASE)
#undef HMM_CASE
  }
  return hipErrorInvalidValue;
}

hipError_t dispatch_fwd(const DevProfile &P, const DevDb &db, const DevOut &o, hipStream_t s) {
  if (coop_instance(P.Q32)) return launch_fwd_coop(P, db, o, s);
  switch (P.Q32) {
#define HMM_CASE(q) \
  case q:           \
    return launch_fwd<q>(P, db, o, s);
    HMM_Q32_CASES(HMM_CASE)
#undef HMM_CASE
  }
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_tail(const DevProfile &P, const DevDb *chunk, int K, const DevOut &o, hipStream_t s,
                       const SearchSync &y, hipEvent_t *ev, bool join = true);

hipError_t launch_search(const DevProfile &P, const DevDb *chunk, int K, const DevOut &o, hipStream_t s,
                         const SearchSync &y, hipEvent_t *ev) {
  if (K < 1 || K > kMaxChunks) return hipErrorInvalidValue;
  hipError_t e = hipSuccess;
  auto ok = [&](hipError_t r) {
    if (e == hipSuccess) e = r;
    return e == hipSuccess;
  };
  auto mark = [&](int i, hipStream_t st) {
    if (ev) ok(hipEventRecord(ev[i], st));
  };
  mark(0, s);
  hipLaunchKernelGGL(clear_counters, dim3(1), dim3(256), 0, s, chunk[0].counters, K);
  ok(hipGetLastError());
  // MSV of every chunk, back to back on the search stream
  for (int k = 0; k < K && e == hipSuccess; k++) {
    if (chunk[k].n > 0) {
      ok(dispatch_msv(P, chunk[k], o, s));
      if (o.bias_filter) ok(launch_bias(P, chunk[k], o, s));
    }
    ok(hipEventRecord(y.msv_done[k], s));
  }
  mark(1, s);
  if (e != hipSuccess) return e;
  return launch_tail(P, chunk, K, o, s, y, ev);
}

// The rest of each chunk's cascade as soon as its MSV is done (event
// y.msv_done[k] on the search stream).  An int16 overflow passes the
// Viterbi filter whatever its exact score, so Forward needs nothing from
// the rescore: the two run side by side.  With `o.fused_tail` and a profile
// that has a fused instance, one kernel takes all three stages instead (the
// rescore stream then has nothing to run).  The counts and the caller-order
// results follow on the tail stream, whose end (y.tail_done) the search
// stream waits for when `join` is set (a group of searches joins them all
// at its end instead).
hipError_t launch_tail(const DevProfile &P, const DevDb *chunk, int K, const DevOut &o, hipStream_t s,
                       const SearchSync &y, hipEvent_t *ev, bool join) {
  hipError_t e = hipSuccess;
  auto ok = [&](hipError_t r) {
    if (e == hipSuccess) e = r;
    return e == hipSuccess;
  };
  auto mark = [&](int i, hipStream_t st) {
    if (ev) ok(hipEventRecord(ev[i], st));
  };
  const bool fused = o.fused_tail && tail_fused_instance(P);
  for (int k = 0; k < K && e == hipSuccess; k++) {
    const bool any = chunk[k].n > 0;
    // the last chunk's stages end the search: their waves take issue
    // priority by target length (an earlier chunk's share the CUs with the
    // next chunk's MSV, which they would hold back)
    DevDb ck = chunk[k];
    ck.prio_by_len = k == K - 1;
    if (!ok(hipStreamWaitEvent(y.tail, y.msv_done[k], 0))) break;
    if (any && !ok(fused ? dispatch_tail_fused(P, ck, o, y.tail) : dispatch_vit16(P, ck, o, y.tail))) break;
    if (!ok(hipEventRecord(y.vit_done[k], y.tail))) break;
    if (k == K - 1) mark(2, y.tail);
    if (!ok(hipStreamWaitEvent(y.aux, y.vit_done[k], 0))) break;
    if (fused) continue;
    if (any && !ok(dispatch_vit32(P, ck, o, y.aux))) break;
    if (any && !ok(dispatch_fwd(P, ck, o, y.tail))) break;
  }
  mark(3, y.aux);
  if (ok(hipEventRecord(y.aux_done, y.aux))) ok(hipStreamWaitEvent(y.tail, y.aux_done, 0));
  if (e == hipSuccess && o.counts) {
    hipLaunchKernelGGL(export_counts, dim3(1), dim3(64), 0, y.tail, (const int32_t *)chunk[0].counters, K,
                       o.counts);
    ok(hipGetLastError());
  }
  // chunk 0 starts at sorted index 0: its sorted arrays are the whole
  // database's
  DevDb all = chunk[0];
  all.n = 0;
  for (int k = 0; k < K; k++) all.n += chunk[k].n;
  if (e == hipSuccess && all.n > 0) {
    hipLaunchKernelGGL(results_kernel, dim3((unsigned)((all.n + 255) / 256)), dim3(256), 0, y.tail, all, o);
    ok(hipGetLastError());
  }
  if (ok(hipEventRecord(y.tail_done, y.tail)) && join) ok(hipStreamWaitEvent(s, y.tail_done, 0));
  if (join) mark(4, s);
  return e;
}

// Several searches of one database (one handle each) by different profiles,
// one chunk each: their counters are cleared, the MSV of profiles sharing a
// diagonal instance runs as group kernels (up to msv_group_max profiles per
// launch; the others alone), then each search's composition-bias filter
// (if on) and its cascade tail on its own handle's streams, all joined back
// into `s`.
hipError_t launch_search_group(const DevProfile *P, const DevDb *db, const DevOut *o, int n, hipStream_t s,
                               const SearchSync *const *y) {
  hipError_t e = hipSuccess;
  auto ok = [&](hipError_t r) {
    if (e == hipSuccess) e = r;
    return e == hipSuccess;
  };
  for (int i = 0; i < n && e == hipSuccess; i++) {
    hipLaunchKernelGGL(clear_counters, dim3(1), dim3(256), 0, s, db[i].counters, 1);
    ok(hipGetLastError());
  }
  std::vector<int> done(n, 0);
  // a search's composition-bias filter (if on) and its cascade tail, on its
  // own handle's streams once its MSV (on `s`) is done
  auto tail = [&](int i) {
    if (o[i].bias_filter && db[i].n > 0) ok(launch_bias(P[i], db[i], o[i], s));
    ok(hipEventRecord(y[i]->msv_done[0], s));
    ok(launch_tail(P[i], &db[i], 1, o[i], s, *y[i], nullptr, false));
  };
  for (int i = 0; i < n && e == hipSuccess; i++) {
    if (done[i] || db[i].n == 0) continue;
    const int gmax = P[i].msv_diag ? msv_group_max(P[i].Qm) : 1;
    std::vector<int> grp{i};
    for (int j = i + 1; j < n && (int)grp.size() < gmax; j++)
      if (!done[j] && P[j].msv_diag && P[j].Qm == P[i].Qm) grp.push_back(j);
    for (int j : grp) done[j] = 1;
    if (grp.size() == 1) {
      ok(dispatch_msv(P[i], db[i], o[i], s));
    } else {
      DevProfile gp[4];
      DevDb gd[4];
      DevOut go[4];
      for (size_t g = 0; g < grp.size(); g++) {
        gp[g] = P[grp[g]];
        gd[g] = db[grp[g]];
        go[g] = o[grp[g]];
      }
      ok(dispatch_msv_group(gp, gd, go, (int)grp.size(), s));
    }
  }
  // The tails start after every MSV launch.  Started right after their own
  // group's launch, they share the CUs with the later MSV launches, which
  // absorb that (their waves take targets from a work counter), but the
  // group still took longer (C4: 350.7 against 345.0 ms).
  for (int i = 0; i < n && e == hipSuccess; i++) tail(i);
  // every search's tail joins the caller's stream
  for (int i = 0; i < n && e == hipSuccess; i++) ok(hipStreamWaitEvent(s, y[i]->tail_done, 0));
  return e;
}

}  // namespace hmmgpu
