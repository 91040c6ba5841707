// HIP kernels (gfx950) of the 32-bit stages for long profiles: Forward (fp32)
// and the exact int32 Viterbi rescore, with one workgroup of W waves per
// target.
//
// With one wave per target, a long profile (Q >= 14 cells per lane and
// state) needs most of the register file for one wave, so a SIMD runs one
// wave and nothing hides its memory and cross-lane latencies.  Here wave w
// of the workgroup holds vectors q in [w*QW, (w+1)*QW) of every lane (cell
// = lane*Q + q, Q = W*QW): the cells of a lane form W consecutive segments,
// one per wave, and several workgroups share a CU.
//
// One barrier per row.  Before it, each wave computes its segment's match
// and insert cells, its delete chain A with nothing entering the segment's
// first cell, and publishes for its lane, into the row's half of a
// double-buffered LDS area (row parity: no wave can run two rows ahead of
// another, as every row ends at the barrier):
//   xo: what the segment passes to the next segment's first delete cell
//       when nothing enters its own first cell (last cell's M through M->D
//       and A through D->D into that cell);
//   ml, il, al: its last cell's M, I and A;
//   Forward: once per wave, the sum of its cells' M g over every lane (its
//   part of E; the exit weight g of a cell carries the deletes it reaches,
//   see hmm_profile_upload);
//   rescore: its running maximum if it crossed the trigger line.
// After the barrier every wave composes its lane's W segment maps
// (x_out = xo + p x_in: affine for Forward, max-plus for the rescore), chains
// the lanes with a DPP prefix scan, and so knows the value x_j entering every
// segment j of its lane.  Its own delete cells are then D_q = A_q (+) P_q
// x_w; Forward's E is the sum of the W published parts; the left
// neighbour of its first cell for the next row (segment w-1 of the lane, or
// segment W-1 of the previous lane through a DPP shift) is (ml, il,
// al (+) P_last x).  All waves hold the same special states and take the
// same decisions.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>

#include "hmm_device.h"
#include "hmm_internal.h"

namespace hmmgpu {
namespace {

// Inclusive prefix scan across lanes (lane l-1 -> l) of affine maps
// x -> a + P x, with the P parts before each step in ps.  A lane without a
// source reads 0 (bound_ctrl), which leaves its map unchanged, so each
// step can be one fused DPP multiply-add.
template <int CTRL, int ROWMASK>
__device__ __forceinline__ float dpp_f0(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, ROWMASK, 0xf, true));
}
__device__ __forceinline__ float affine_scan(float a, const float (&ps)[6]) {
  a = fmaf(dpp_f0<kRowShr1, 0xf>(a), ps[0], a);
  a = fmaf(dpp_f0<kRowShr2, 0xf>(a), ps[1], a);
  a = fmaf(dpp_f0<kRowShr4, 0xf>(a), ps[2], a);
  a = fmaf(dpp_f0<kRowShr8, 0xf>(a), ps[3], a);
  a = fmaf(dpp_f0<kRowBcast15, 0xa>(a), ps[4], a);
  a = fmaf(dpp_f0<kRowBcast31, 0xc>(a), ps[5], a);
  return a;
}
__device__ __forceinline__ void affine_steps(float p, float (&ps)[6]) {
  ps[0] = p;
  p = p * dpp_f<kRowShr1, 0xf>(p, 1.0f);
  ps[1] = p;
  p = p * dpp_f<kRowShr2, 0xf>(p, 1.0f);
  ps[2] = p;
  p = p * dpp_f<kRowShr4, 0xf>(p, 1.0f);
  ps[3] = p;
  p = p * dpp_f<kRowShr8, 0xf>(p, 1.0f);
  ps[4] = p;
  p = p * dpp_f<kRowBcast15, 0xa>(p, 1.0f);
  ps[5] = p;
}

// int32 max-plus maps x -> max(a, x + b) of the rescore's delete chain.
// Their slopes b (profile constants, composed once per kernel) treat a b at
// or below kNeg32 as minus infinity (a structural entry: no delete
// transition into cell 0 or into padding cells), and sums involving it stay
// at kNeg32; every other b is a sum of at most 3071 transition scores
// >= -32768, so no sum leaves int32 and every composed b is >= -2^30.
__device__ __forceinline__ int ninf_add(int x, int b) { return (x <= kNeg32 || b <= kNeg32) ? kNeg32 : x + b; }

template <int CTRL, int ROWMASK>
__device__ __forceinline__ int dpp_i(int v, int fill) {
  return __builtin_amdgcn_update_dpp(fill, v, CTRL, ROWMASK, 0xf, false);
}
// The per-row scan: every map value is at or above the delete floor tau >=
// -2^30 and every composed b at or above -2^30 (see the rescore kernel), so
// plain adds cannot leave int32 and a sum with a minus-infinity b stays
// below the floor, where the maximum with the lane's own value drops it.
__device__ __forceinline__ int maxplus_scan_i(int a, const int (&bs)[6]) {
  a = max(a, dpp_i<kRowShr1, 0xf>(a, kNeg32) + bs[0]);
  a = max(a, dpp_i<kRowShr2, 0xf>(a, kNeg32) + bs[1]);
  a = max(a, dpp_i<kRowShr4, 0xf>(a, kNeg32) + bs[2]);
  a = max(a, dpp_i<kRowShr8, 0xf>(a, kNeg32) + bs[3]);
  a = max(a, dpp_i<kRowBcast15, 0xa>(a, kNeg32) + bs[4]);
  a = max(a, dpp_i<kRowBcast31, 0xc>(a, kNeg32) + bs[5]);
  return a;
}
__device__ __forceinline__ void maxplus_steps_i(int b, int (&bs)[6]) {
  bs[0] = b;
  b = ninf_add(b, dpp_i<kRowShr1, 0xf>(b, 0));
  bs[1] = b;
  b = ninf_add(b, dpp_i<kRowShr2, 0xf>(b, 0));
  bs[2] = b;
  b = ninf_add(b, dpp_i<kRowShr4, 0xf>(b, 0));
  bs[3] = b;
  b = ninf_add(b, dpp_i<kRowShr8, 0xf>(b, 0));
  bs[4] = b;
  b = ninf_add(b, dpp_i<kRowBcast15, 0xa>(b, 0));
  bs[5] = b;
}

__device__ __forceinline__ int fl32(int v) { return max(v, kNeg32); }

// The workgroup's next target (thread 0 takes it from the work counter).
__device__ __forceinline__ int next_target(int32_t *work, int *slot) {
  __syncthreads();
  if (threadIdx.x == 0) *slot = atomicAdd(work, 1);
  __syncthreads();
  return __builtin_amdgcn_readfirstlane(*slot);
}

// ============================================================================ Forward
template <int W>
struct FwdCoopLds {
  float xo[2][W][kWave], ml[2][W][kWave], il[2][W][kWave], al[2][W][kWave], es[2][W];
  int slot;
};

// The work of wave WI of a Forward workgroup (its segment index a
// constant): every wave runs its own instance, and all instances take the
// same barriers in the same order.
template <int QW, int W, int WI>
__device__ __forceinline__ void fwd_coop_wave(const DevProfile &P, const DevDb &db, const DevOut &out,
                                              FwdCoopLds<W> &sh) {
  constexpr int Q = QW * W;
  constexpr int w = WI;
  constexpr int q0 = w * QW;
  constexpr int nb = w > 0 ? w - 1 : W - 1;   // segment of the first cell's left neighbour
  auto &sxo = sh.xo;
  auto &sml = sh.ml;
  auto &sil = sh.il;
  auto &sal = sh.al;
  auto &ses = sh.es;
  const int lane = threadIdx.x & 63;
  const float *trg = P.f_tr + lane;
  // transition planes of this wave's cells, registers
  float tr[TR_N][QW];
#pragma unroll
  for (int k = 0; k < TR_N; k++)
#pragma unroll
    for (int q = 0; q < QW; q++) tr[k][q] = trg[(k * Q + q0 + q) * kWave];
  // transition of `plane` into the first cell after segment j (this lane's
  // segment j + 1, or the next lane's first cell; probability 0 at the end)
  auto into_next = [&](int plane, int j) -> float {
    if (j + 1 < W) return trg[(plane * Q + (j + 1) * QW) * kWave];
    return lane + 1 < kWave ? trg[plane * Q * kWave + 1] : 0.0f;
  };
  // exit weights of this wave's cells: a row's E = sum over cells of M g
  // (the delete cells' part included through g)
  float gx[QW];
#pragma unroll
  for (int q = 0; q < QW; q++) gx[q] = trg[(TR_EXIT * Q + q0 + q) * kWave];
  // pre[q]: product of DD over this wave's cells 1..q; per segment j of the
  // lane: pl[j] the product over its cells 1..QW-1, pj[j] = pl[j] DD' (its
  // map's slope); the lane map slope's scan steps
  float pre[QW], pl[W], pj[W], ps[6];
  {
    float acc = 1.0f;
#pragma unroll
    for (int q = 0; q < QW; q++) {
      if (q) acc *= tr[TR_DDIN][q];
      pre[q] = acc;
    }
    float lanep = 1.0f;
#pragma unroll
    for (int j = 0; j < W; j++) {
      float a = 1.0f;
      for (int q = 1; q < QW; q++) a *= trg[(TR_DDIN * Q + j * QW + q) * kWave];
      pl[j] = a;
      pj[j] = a * into_next(TR_DDIN, j);
      lanep *= pj[j];
    }
    affine_steps(lanep, ps);
  }
  const float mdn = into_next(TR_MDIN, w), ddn = into_next(TR_DDIN, w);
  const float entry_p = P.entry_p;
  const int count = uni(__atomic_load_n(&db.counters[CNT_FWD], __ATOMIC_RELAXED));
  for (;;) {
    const int idx = next_target(&db.counters[CNT_WORK_FWD], &sh.slot);
    if (idx >= count) break;
    const int t = uni(db.list_fwd[idx]);
    const int L = uni(db.len[t]);
    const LenParams lp = db.lp[L];
    const float loop = lp.loop_p, move = lp.move_p;
    float M[QW], I[QW], D[QW];
#pragma unroll
    for (int q = 0; q < QW; q++) M[q] = I[q] = D[q] = 0.0f;
    float pM = 0.0f, pI = 0.0f, pD = 0.0f;   // previous row, left neighbour of the first cell
    float N = 1.0f, B = move, J = 0.0f, C = 0.0f;
    int shift = 0, par = 0;
    // row of residue a: a wave-uniform base (scalar address) and the lane
    // as the only vector part of every read
    auto load = [&](float(&e)[2 * QW], int a) {
      const float *em = P.f_emit + (size_t)a * (2 * Q * kWave) + q0 * kWave;
#pragma unroll
      for (int q = 0; q < QW; q++) {
        e[q] = em[q * kWave + lane];
        e[QW + q] = em[(Q + q) * kWave + lane];
      }
    };
    auto row = [&](const float(&em)[2 * QW]) -> bool {
      const float bent = B * entry_p;
#pragma unroll
      for (int q = QW - 1; q >= 0; q--) {
        const float pm = q ? M[q - 1] : pM, pi = q ? I[q - 1] : pI, pd = q ? D[q - 1] : pD;
        const float sm = fmaf(pm, tr[TR_MMIN][q], fmaf(pi, tr[TR_IMIN][q], fmaf(pd, tr[TR_DMIN][q], bent)));
        const float si = fmaf(M[q], tr[TR_MI][q], I[q] * tr[TR_II][q]);
        M[q] = em[q] * sm;
        I[q] = em[QW + q] * si;
      }
      // this wave's part of E (every lane's segment), reduced before the
      // barrier: it needs no delete value, so its cross-lane sum overlaps
      // the delete chain below instead of following the barrier
      float es = 0.0f;
#pragma unroll
      for (int q = 0; q < QW; q++) es = fmaf(M[q], gx[q], es);
      es = wave_sum_fused(es);
      // delete chain with nothing entering the segment (A)
      D[0] = 0.0f;
#pragma unroll
      for (int q = 1; q < QW; q++) D[q] = fmaf(M[q - 1], tr[TR_MDIN][q], D[q - 1] * tr[TR_DDIN][q]);
      sxo[par][w][lane] = fmaf(M[QW - 1], mdn, D[QW - 1] * ddn);
      sml[par][w][lane] = M[QW - 1];
      sil[par][w][lane] = I[QW - 1];
      sal[par][w][lane] = D[QW - 1];
      if (lane == 0) ses[par][w] = es;
      __syncthreads();
      // the values entering the lane's segments
      float a = sxo[par][0][lane];
#pragma unroll
      for (int j = 1; j < W; j++) a = fmaf(pj[j], a, sxo[par][j][lane]);
      float x = lane_up_f(affine_scan_fused(a, ps));
      float xw = x, xn = x, E = ses[par][0];
#pragma unroll
      for (int j = 0; j < W; j++) {
        if (j == w) xw = x;
        if (j == nb) xn = x;
        if (j) E += ses[par][j];
        if (j + 1 < W) x = fmaf(pj[j], x, sxo[par][j][lane]);
      }
#pragma unroll
      for (int q = 0; q < QW; q++) D[q] = fmaf(pre[q], xw, D[q]);
      // the first cell's left neighbour for the next row
      pM = sml[par][nb][lane];
      pI = sil[par][nb][lane];
      pD = fmaf(pl[nb], xn, sal[par][nb][lane]);
      if constexpr (w == 0) {
        pM = lane_up_f(pM);
        pI = lane_up_f(pI);
        pD = lane_up_f(pD);
      }
      par ^= 1;
      E = __builtin_bit_cast(float, uni(__builtin_bit_cast(int, E)));
      J = fmaf(J, loop, 0.5f * E);
      C = fmaf(C, loop, 0.5f * E);
      N = N * loop;
      B = (N + J) * move;
      const float big = fmaxf(fmaxf(fmaxf(E, J), fmaxf(C, N)), B);
      if (big > 0x1p40f || big < 0x1p-40f) {
        int ex;
        (void)frexpf(big, &ex);
        ex = uni(ex);
        const float sc = ldexpf(1.0f, -ex);
#pragma unroll
        for (int q = 0; q < QW; q++) {
          M[q] *= sc;
          I[q] *= sc;
          D[q] *= sc;
        }
        pM *= sc;
        pI *= sc;
        pD *= sc;
        J *= sc;
        C *= sc;
        N *= sc;
        B *= sc;
        shift += ex;
      }
      return false;
    };
    float ea[2 * QW], eb[2 * QW];
    int stop;
    (void)drive_rows(db.res + db.start[t], L, 0, 0, stop, lane, ea, eb, load, row);
    if constexpr (w == 0) {
      const float f = (float)(log((double)C * (double)move) + (double)shift * M_LN2);
      const bool pass = f > lp.fthr;
      const uint8_t fl = (uint8_t)(uni(db.flags_sorted[t]) | HMM_FWD_RAN | (pass ? HMM_FWD_PASS : 0));
      db.flags_sorted[t] = fl;
      out.fwd[uni(db.perm[t])] = f;
      if (pass) (void)wave_fetch_add(&db.counters[CNT_FWD_PASS], 1);
    }
  }
}



template <int QW, int W>
__global__ void __launch_bounds__(64 * W) fwd_coop_kernel(DevProfile P, DevDb db, DevOut out) {
  static_assert(W == 2 || W == 4, "two or four waves per target");
  __shared__ FwdCoopLds<W> sh;
  const int w = (int)__builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  if (w == 0) {
    fwd_coop_wave<QW, W, 0>(P, db, out, sh);
  } else if (w == 1) {
    fwd_coop_wave<QW, W, 1>(P, db, out, sh);
  } else if constexpr (W == 4) {
    if (w == 2)
      fwd_coop_wave<QW, W, 2>(P, db, out, sh);
    else
      fwd_coop_wave<QW, W, 3>(P, db, out, sh);
  }
}

// ============================================================================ int32 rescore
//
// The delete floor of the one-wave kernels: the chain keeps D' = max(D,
// tau), tau = xBe - max_k DM_k >= -2^30, which changes no match cell (a
// delete value at or below tau enters a match cell at or below xBe, which
// every match cell already includes).  With it the segment maps are exact
// in plain int32 adds:
//   - inside a segment D'_q = max(M_{q-1} + MD, D'_{q-1} + DD, tau), from
//     D'_0 = tau with nothing entering; the value x entering the first cell
//     then gives D'_q = max(A_q, x + pre_q), and the next segment receives
//     max(xo, x + pj) with xo >= tau;
//   - every operand of an add is >= -2^30 (states, floors, table entries
//     and the composed b, which are exact DD sums >= -3072 * 32768 or the
//     structural -2^30), so no add leaves int32;
//   - a sum with a structural -2^30 is at most (largest score) - 2^30, below
//     tau >= -2^17 while every score stays below 2^29 (the host rejects a
//     search whose longest target times largest emission score could reach
//     that), and each such sum meets a maximum with a term >= tau, so it
//     is dropped exactly as minus infinity would be.
// Lane l receives lane l-1's value; lane 0 receives `fill`.
__device__ __forceinline__ int lane_up_fill(int v, int fill) {
  return __builtin_amdgcn_update_dpp(fill, v, 0x138 /* wave_shr:1 */, 0xf, 0xf, false);
}

template <int W>
struct VitCoopLds {
  int xo[2][W][kWave], ml[2][W][kWave], il[2][W][kWave], al[2][W][kWave];
  int xs[2][W];   // per wave: its maximum when it crossed the trigger line, else kNeg32
  int fin[W];
  int slot;
};

// The work of wave WI of a rescore workgroup, as in the Forward kernel.
template <int QW, int W, int WI>
__device__ __forceinline__ void vit32_coop_wave(const DevProfile &P, const DevDb &db, const DevOut &out,
                                                VitCoopLds<W> &sh) {
  constexpr int Q = QW * W;
  constexpr int w = WI;
  constexpr int q0 = w * QW;
  constexpr int nb = w > 0 ? w - 1 : W - 1;
  auto &sxo = sh.xo;
  auto &sml = sh.ml;
  auto &sil = sh.il;
  auto &sal = sh.al;
  auto &sxs = sh.xs;
  auto &fin = sh.fin;
  const int lane = threadIdx.x & 63;
  const int *trg = P.v32_tr + lane;
  int tr[TR_N][QW];
#pragma unroll
  for (int k = 0; k < TR_N; k++)
#pragma unroll
    for (int q = 0; q < QW; q++) tr[k][q] = trg[(k * Q + q0 + q) * kWave];
  auto into_next = [&](int plane, int j) -> int {
    if (j + 1 < W) return trg[(plane * Q + (j + 1) * QW) * kWave];
    return lane + 1 < kWave ? trg[plane * Q * kWave + 1] : kNeg32;
  };
  // max-plus counterparts of the Forward kernel's products: sums of DD
  // (minus infinity absorbing) over cells 1..q of this wave, over cells
  // 1..QW-1 of each segment (pl), plus DD' (pj); the lane map's scan steps
  int pre[QW], pl[W], pj[W], bs[6];
  {
    int acc = 0;
#pragma unroll
    for (int q = 0; q < QW; q++) {
      if (q) acc = ninf_add(acc, tr[TR_DDIN][q]);
      pre[q] = acc;
    }
    int lanep = 0;
#pragma unroll
    for (int j = 0; j < W; j++) {
      int a = 0;
      for (int q = 1; q < QW; q++) a = ninf_add(a, trg[(TR_DDIN * Q + j * QW + q) * kWave]);
      pl[j] = a;
      pj[j] = ninf_add(a, into_next(TR_DDIN, j));
      lanep = ninf_add(lanep, pj[j]);
    }
    maxplus_steps_i(lanep, bs);
  }
  const int mdn = into_next(TR_MDIN, w), ddn = into_next(TR_DDIN, w);
  const int count = uni(__atomic_load_n(&db.counters[CNT_OVF], __ATOMIC_RELAXED));
  for (;;) {
    const int idx = next_target(&db.counters[CNT_WORK_OVF], &sh.slot);
    if (idx >= count) break;
    const int t = uni(db.list_ovf[idx]);
    const int L = uni(db.len[t]);
    const LenParams lp = db.lp[L];
    const int mv = lp.move16, ej = P.ej16, entry = P.entry16;
    int M[QW], I[QW], D[QW];
#pragma unroll
    for (int q = 0; q < QW; q++) M[q] = I[q] = D[q] = kNeg32;
    int pM = kNeg32, pI = kNeg32, pD = kNeg32;
    int accM = kNeg32, xJt = kNeg32;
    int xbe = fl32(fl32(mv) + entry);
    int tau = xbe - P.dm_max32;   // delete floor
    int T = -ej + 1;
    int par = 0;
    auto load = [&](int(&e)[2 * QW], int a) {
      const int *em = P.v32_emit + (size_t)a * (2 * Q * kWave) + q0 * kWave;
#pragma unroll
      for (int q = 0; q < QW; q++) {
        e[q] = em[q * kWave + lane];
        e[QW + q] = em[(Q + q) * kWave + lane];
      }
    };
    auto row = [&](const int(&em)[2 * QW]) -> bool {
      // saturating adds and two floors, as in the one-wave kernel: a match
      // or insert value below -2^30 only meets maxima with a term >= -2^30
      // (xBe, the insert floor, tau); the value shifted into cell 0 is
      // irrelevant, as every transition into it is kNeg32
#pragma unroll
      for (int q = QW - 1; q >= 0; q--) {
        const int pm = q ? M[q - 1] : pM, pi = q ? I[q - 1] : pI, pd = q ? D[q - 1] : pD;
        const int m = max(max(xbe, sadd32(pm, tr[TR_MMIN][q])),
                          max(sadd32(pi, tr[TR_IMIN][q]), sadd32(pd, tr[TR_DMIN][q])));
        const int mn = sadd32(m, em[q]);
        const int in =
            sadd32(max(max(sadd32(M[q], tr[TR_MI][q]), sadd32(I[q], tr[TR_II][q])), kNeg32), em[QW + q]);
        accM = max(accM, mn);
        M[q] = mn;
        I[q] = in;
      }
      // delete chain with only the floor entering the segment
      D[0] = tau;
#pragma unroll
      for (int q = 1; q < QW; q++)
        D[q] = max(max(sadd32(M[q - 1], tr[TR_MDIN][q]), D[q - 1] + tr[TR_DDIN][q]), tau);
      sxo[par][w][lane] = max(max(sadd32(M[QW - 1], mdn), D[QW - 1] + ddn), tau);
      sml[par][w][lane] = M[QW - 1];
      sil[par][w][lane] = I[QW - 1];
      sal[par][w][lane] = D[QW - 1];
      // some cell reached the line that could raise xJ: its wave's maximum
      const bool trig = __builtin_amdgcn_ballot_w64(accM >= T) != 0;
      const int wm = trig ? wave_max_i32(accM) : kNeg32;
      if (lane == 0) sxs[par][w] = wm;
      __syncthreads();
      int a = sxo[par][0][lane];
#pragma unroll
      for (int j = 1; j < W; j++) a = max(sxo[par][j][lane], a + pj[j]);
      int x = lane_up_fill(maxplus_scan_i(a, bs), tau);
      int xw = x, xn = x;
#pragma unroll
      for (int j = 0; j < W; j++) {
        if (j == w) xw = x;
        if (j == nb) xn = x;
        if (j + 1 < W) x = max(sxo[par][j][lane], x + pj[j]);
      }
#pragma unroll
      for (int q = 0; q < QW; q++) D[q] = max(D[q], xw + pre[q]);
      pM = sml[par][nb][lane];
      pI = sil[par][nb][lane];
      pD = max(sal[par][nb][lane], xn + pl[nb]);
      if constexpr (w == 0) {
        pM = lane_up_fill(pM, kNeg32);
        pI = lane_up_fill(pI, kNeg32);
        pD = lane_up_fill(pD, kNeg32);
      }
      int m = kNeg32;
#pragma unroll
      for (int j = 0; j < W; j++) m = max(m, sxs[par][j]);
      par ^= 1;
      if (m > kNeg32) {
        xJt = max(xJt, fl32(m + ej));
        const int xB = max(fl32(mv), fl32(xJt + mv));
        xbe = fl32(xB + entry);
        tau = xbe - P.dm_max32;
        T = max(xJt, 0) - ej + 1;
      }
      return false;
    };
    int ea[2 * QW], eb[2 * QW];
    int stop;
    (void)drive_rows(db.res + db.start[t], L, 0, 0, stop, lane, ea, eb, load, row);
    // the final maximum over every cell of every row, all waves
    {
      const int v = wave_max_i32(accM);
      if (lane == 0) fin[w] = v;
      __syncthreads();
      int m = kNeg32;
#pragma unroll
      for (int j = 0; j < W; j++) m = max(m, fin[j]);
      if constexpr (w == 0) out.vit[uni(db.perm[t])] = fl32(fl32(m + ej) + mv);
    }
  }
}

template <int QW, int W>
__global__ void __launch_bounds__(64 * W) vit32_coop_kernel(DevProfile P, DevDb db, DevOut out) {
  static_assert(W == 2 || W == 4, "two or four waves per target");
  __shared__ VitCoopLds<W> sh;
  const int w = (int)__builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  if (w == 0) {
    vit32_coop_wave<QW, W, 0>(P, db, out, sh);
  } else if (w == 1) {
    vit32_coop_wave<QW, W, 1>(P, db, out, sh);
  } else if constexpr (W == 4) {
    if (w == 2)
      vit32_coop_wave<QW, W, 2>(P, db, out, sh);
    else
      vit32_coop_wave<QW, W, 3>(P, db, out, sh);
  }
}

template <int QW, int W, typename K>
hipError_t launch_coop(K k, int &bpc, const DevProfile &P, const DevDb &db, const DevOut &o, hipStream_t s) {
  constexpr int threads = 64 * W;
  if (!bpc) {
    int nb = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, k, threads, 0) != hipSuccess || nb < 1) nb = 1;
    bpc = nb;
  }
  int dev = 0, ncu = 0;
  (void)hipGetDevice(&dev);
  (void)hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev);
  if (ncu <= 0) ncu = 256;
  int64_t blocks = (int64_t)bpc * ncu;
  if (blocks > db.n) blocks = db.n;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k, dim3((unsigned)blocks), dim3(threads), 0, s, P, db, o);
  return hipGetLastError();
}

}  // namespace

// Q -> (QW, W): two waves for 14 vectors per lane, four from 16 on.
#define HMM_COOP_CASES(X) X(14, 7, 2) X(16, 4, 4) X(20, 5, 4) X(24, 6, 4) X(28, 7, 4) X(32, 8, 4) X(40, 10, 4) X(48, 12, 4)

bool coop_instance(int Q) {
  switch (Q) {
#define HMM_CASE(q, qw, w) \
  case q:                  \
    return true;
    HMM_COOP_CASES(HMM_CASE)
#undef HMM_CASE
  }
  return false;
}

hipError_t launch_fwd_coop(const DevProfile &P, const DevDb &db, const DevOut &o, hipStream_t s) {
  switch (P.Q32) {
#define HMM_CASE(q, qw, w)                                                      \
  case q: {                                                                     \
    static int bpc = 0;                                                         \
    return launch_coop<qw, w>(fwd_coop_kernel<qw, w>, bpc, P, db, o, s);        \
  }
    HMM_COOP_CASES(HMM_CASE)
#undef HMM_CASE
  }
  return hipErrorInvalidValue;
}

hipError_t launch_vit32_coop(const DevProfile &P, const DevDb &db, const DevOut &o, hipStream_t s) {
  switch (P.Q32) {
#define HMM_CASE(q, qw, w)                                                      \
  case q: {                                                                     \
    static int bpc = 0;                                                         \
    return launch_coop<qw, w>(vit32_coop_kernel<qw, w>, bpc, P, db, o, s);      \
  }
    HMM_COOP_CASES(HMM_CASE)
#undef HMM_CASE
  }
  return hipErrorInvalidValue;
}

}  // namespace hmmgpu
