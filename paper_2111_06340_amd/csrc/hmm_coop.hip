// HIP kernels (gfx950) of the 32-bit stages for long profiles: Forward (fp32)
// and the exact int32 Viterbi rescore, with one workgroup of W waves per
// target.
//
// With one wave per target, a long profile (Q >= 14 cells per lane and
// state) needs most of the register file for one wave, so a SIMD runs one
// wave and nothing hides its memory and cross-lane latencies.  Here wave w
// of the workgroup holds vectors q in [w*QW, (w+1)*QW) of every lane (cell
// = lane*Q + q, Q = W*QW), so each wave carries a quarter of the state and
// several workgroups share a CU.  Per row, through a few hundred bytes of
// LDS and three barriers, the waves exchange:
//   - the previous row's M, I, D of each wave's last cell (the left
//     neighbour of the next wave's first cell; wave 0 takes wave W-1's of
//     the previous lane);
//   - the current row's M of each wave's last cell (input of the next
//     wave's first delete cell);
//   - each wave's delete-chain map over its cells with zero entry value:
//     the lane's map is their composition, the lanes are then chained by a
//     DPP prefix scan (affine maps x -> a + P x for Forward, max-plus maps
//     x -> max(a, x + b) for the rescore), and each wave applies the value
//     entering its first cell;
//   - each wave's part of E (Forward: a sum) or of the running maximum
//     (rescore: only when it crossed the line that could change xJ).
// All waves then hold the same special states and take the same decisions.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>

#include "hmm_device.h"
#include "hmm_internal.h"

namespace hmmgpu {
namespace {

// Inclusive prefix scan across lanes (lane l-1 -> l) of affine maps
// x -> a + P x, with the P parts before each step in ps.
__device__ __forceinline__ float affine_scan(float a, const float (&ps)[6]) {
  a = fmaf(ps[0], dpp_f<kRowShr1, 0xf>(a, 0.0f), a);
  a = fmaf(ps[1], dpp_f<kRowShr2, 0xf>(a, 0.0f), a);
  a = fmaf(ps[2], dpp_f<kRowShr4, 0xf>(a, 0.0f), a);
  a = fmaf(ps[3], dpp_f<kRowShr8, 0xf>(a, 0.0f), a);
  a = fmaf(ps[4], dpp_f<kRowBcast15, 0xa>(a, 0.0f), a);
  a = fmaf(ps[5], dpp_f<kRowBcast31, 0xc>(a, 0.0f), a);
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

// int32 max-plus maps x -> max(a, x + b) of the rescore's delete chain.  A
// value or a b at or below kNeg32 is minus infinity (a structural entry:
// no delete transition into cell 0 or into padding cells), and sums
// involving it stay there; every other b is a sum of at most 3071
// transition scores >= -32768, so no sum leaves int32.
__device__ __forceinline__ int ninf_add(int x, int b) { return (x <= kNeg32 || b <= kNeg32) ? kNeg32 : x + b; }

template <int CTRL, int ROWMASK>
__device__ __forceinline__ int dpp_i(int v, int fill) {
  return __builtin_amdgcn_update_dpp(fill, v, CTRL, ROWMASK, 0xf, false);
}
__device__ __forceinline__ int maxplus_scan_i(int a, const int (&bs)[6]) {
  a = max(a, ninf_add(dpp_i<kRowShr1, 0xf>(a, kNeg32), bs[0]));
  a = max(a, ninf_add(dpp_i<kRowShr2, 0xf>(a, kNeg32), bs[1]));
  a = max(a, ninf_add(dpp_i<kRowShr4, 0xf>(a, kNeg32), bs[2]));
  a = max(a, ninf_add(dpp_i<kRowShr8, 0xf>(a, kNeg32), bs[3]));
  a = max(a, ninf_add(dpp_i<kRowBcast15, 0xa>(a, kNeg32), bs[4]));
  a = max(a, ninf_add(dpp_i<kRowBcast31, 0xc>(a, kNeg32), bs[5]));
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
template <int QW, int W>
__global__ void __launch_bounds__(64 * W) fwd_coop_kernel(DevProfile P, DevDb db, DevOut out) {
  constexpr int Q = QW * W;
  __shared__ float bM[W][kWave], bI[W][kWave], bD[W][kWave];   // previous row, last cell of each wave
  __shared__ float cM[W][kWave];                                // current row M, last cell of each wave
  __shared__ float mA[W][kWave];                                // delete chain with zero entry, last cell
  __shared__ float eS[W];                                       // parts of E
  __shared__ int slot;
  const int lane = threadIdx.x & 63;
  const int w = (int)__builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int q0 = w * QW;
  const float *trg = P.f_tr + lane;
  // transition planes of this wave's cells, registers
  float tr[TR_N][QW];
#pragma unroll
  for (int k = 0; k < TR_N; k++)
#pragma unroll
    for (int q = 0; q < QW; q++) tr[k][q] = trg[(k * Q + q0 + q) * kWave];
  // delete chain products: inside this wave up to q, over each wave's cells
  // of this lane, over the whole lane, and the lane scan's steps
  float pre[QW], pw[W], ps[6];
  {
    float acc = 1.0f;
#pragma unroll
    for (int q = 0; q < QW; q++) {
      acc *= tr[TR_DDIN][q];
      pre[q] = acc;
    }
    float pl = 1.0f;
#pragma unroll
    for (int j = 0; j < W; j++) {
      float pj = 1.0f;
      for (int q = 0; q < QW; q++) pj *= trg[(TR_DDIN * Q + j * QW + q) * kWave];
      pw[j] = pj;
      pl *= pj;
    }
    affine_steps(pl, ps);
  }
  const float entry_p = P.entry_p;
  const float *emit = P.f_emit + lane;
  const int count = uni(__atomic_load_n(&db.counters[CNT_FWD], __ATOMIC_RELAXED));
  for (;;) {
    const int idx = next_target(&db.counters[CNT_WORK_FWD], &slot);
    if (idx >= count) break;
    const int t = uni(db.list_fwd[idx]);
    const int L = uni(db.len[t]);
    const LenParams lp = db.lp[L];
    const float loop = lp.loop_p, move = lp.move_p;
    float M[QW], I[QW], D[QW];
#pragma unroll
    for (int q = 0; q < QW; q++) M[q] = I[q] = D[q] = 0.0f;
    bM[w][lane] = bI[w][lane] = bD[w][lane] = 0.0f;
    __syncthreads();
    float N = 1.0f, B = move, J = 0.0f, C = 0.0f;
    int shift = 0;
    auto load = [&](float(&e)[2 * QW], int a) {
      const float *er = emit + a * (2 * Q * kWave);
#pragma unroll
      for (int q = 0; q < QW; q++) {
        e[q] = er[(q0 + q) * kWave];
        e[QW + q] = er[(Q + q0 + q) * kWave];
      }
    };
    auto row = [&](const float(&em)[2 * QW]) -> bool {
      // left neighbours (previous row) of this wave's first cell
      const int wl = w > 0 ? w - 1 : W - 1;
      const int ll = w > 0 ? lane : lane - 1;
      const float pM = ll >= 0 ? bM[wl][max(ll, 0)] : 0.0f, pI = ll >= 0 ? bI[wl][max(ll, 0)] : 0.0f,
                  pD = ll >= 0 ? bD[wl][max(ll, 0)] : 0.0f;
      const float bent = B * entry_p;
#pragma unroll
      for (int q = QW - 1; q >= 0; q--) {
        const float pm = q ? M[q - 1] : pM, pi = q ? I[q - 1] : pI, pd = q ? D[q - 1] : pD;
        const float sm = fmaf(pm, tr[TR_MMIN][q], fmaf(pi, tr[TR_IMIN][q], fmaf(pd, tr[TR_DMIN][q], bent)));
        const float si = fmaf(M[q], tr[TR_MI][q], I[q] * tr[TR_II][q]);
        M[q] = em[q] * sm;
        I[q] = em[QW + q] * si;
      }
      cM[w][lane] = M[QW - 1];
      __syncthreads();   // B1: current-row boundary M
      const float cin = ll >= 0 ? cM[wl][max(ll, 0)] : 0.0f;
      float dc = 0.0f;
#pragma unroll
      for (int q = 0; q < QW; q++) {
        D[q] = fmaf(q ? M[q - 1] : cin, tr[TR_MDIN][q], dc * tr[TR_DDIN][q]);
        dc = D[q];
      }
      mA[w][lane] = D[QW - 1];
      __syncthreads();   // B2: delete-chain maps
      float a = 0.0f, cw = 0.0f;
#pragma unroll
      for (int j = 0; j < W; j++) a = fmaf(pw[j], a, mA[j][lane]);
      const float lane_in = lane_up_f(affine_scan(a, ps));
      cw = lane_in;
      for (int j = 0; j < w; j++) cw = fmaf(pw[j], cw, mA[j][lane]);
      float part = 0.0f;
#pragma unroll
      for (int q = 0; q < QW; q++) {
        D[q] = fmaf(cw, pre[q], D[q]);
        part += M[q] + D[q];
      }
      const float ws = wave_sum_f(part);
      if (lane == 0) eS[w] = ws;
      bM[w][lane] = M[QW - 1];
      bI[w][lane] = I[QW - 1];
      bD[w][lane] = D[QW - 1];
      __syncthreads();   // B3: E parts and the next row's boundaries
      float E = 0.0f;
#pragma unroll
      for (int j = 0; j < W; j++) E += eS[j];
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
        for (int q = 0; q < QW; q++) {
          M[q] *= s;
          I[q] *= s;
          D[q] *= s;
        }
        J *= s;
        C *= s;
        N *= s;
        B *= s;
        shift += ex;
        // the stored boundaries are read after the next B3 only for the
        // row after next; the next row reads them scaled:
        bM[w][lane] = M[QW - 1];
        bI[w][lane] = I[QW - 1];
        bD[w][lane] = D[QW - 1];
        __syncthreads();   // every wave takes the same branch
      }
      return false;
    };
    float ea[2 * QW], eb[2 * QW];
    int stop;
    (void)drive_rows(db.res + db.start[t], L, 0, 0, stop, lane, ea, eb, load, row);
    if (w == 0) {
      const float f = (float)(log((double)C * (double)move) + (double)shift * M_LN2);
      const bool pass = f > lp.fthr;
      const uint8_t fl = (uint8_t)(uni(db.flags_sorted[t]) | HMM_FWD_RAN | (pass ? HMM_FWD_PASS : 0));
      const int c = uni(db.perm[t]);
      out.fwd[c] = f;
      out.flags[c] = fl;
      if (pass) (void)wave_fetch_add(&db.counters[CNT_FWD_PASS], 1);
    }
  }
}

// ============================================================================ int32 rescore
template <int QW, int W>
__global__ void __launch_bounds__(64 * W) vit32_coop_kernel(DevProfile P, DevDb db, DevOut out) {
  constexpr int Q = QW * W;
  __shared__ int bM[W][kWave], bI[W][kWave], bD[W][kWave];
  __shared__ int cM[W][kWave];
  __shared__ int mA[W][kWave];
  __shared__ int xS[W];        // per wave: its maximum when it crossed the trigger line, else kNeg32
  __shared__ int slot;
  const int lane = threadIdx.x & 63;
  const int w = (int)__builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int q0 = w * QW;
  const int *trg = P.v32_tr + lane;
  int tr[TR_N][QW];
#pragma unroll
  for (int k = 0; k < TR_N; k++)
#pragma unroll
    for (int q = 0; q < QW; q++) tr[k][q] = trg[(k * Q + q0 + q) * kWave];
  // delete chain sums (max-plus b parts): inside this wave up to q, over each
  // wave's cells of this lane, over the lane, and the lane scan's steps
  int pre[QW], bw[W], bs[6];
  {
    int acc = 0;
#pragma unroll
    for (int q = 0; q < QW; q++) {
      acc = ninf_add(acc, tr[TR_DDIN][q]);
      pre[q] = acc;
    }
    int bl = 0;
#pragma unroll
    for (int j = 0; j < W; j++) {
      int bj = 0;
      for (int q = 0; q < QW; q++) bj = ninf_add(bj, trg[(TR_DDIN * Q + j * QW + q) * kWave]);
      bw[j] = bj;
      bl = ninf_add(bl, bj);
    }
    maxplus_steps_i(bl, bs);
  }
  const int *emit = P.v32_emit + lane;
  const int count = uni(__atomic_load_n(&db.counters[CNT_OVF], __ATOMIC_RELAXED));
  for (;;) {
    const int idx = next_target(&db.counters[CNT_WORK_OVF], &slot);
    if (idx >= count) break;
    const int t = uni(db.list_ovf[idx]);
    const int L = uni(db.len[t]);
    const LenParams lp = db.lp[L];
    const int mv = lp.move16, ej = P.ej16, entry = P.entry16;
    int M[QW], I[QW], D[QW];
#pragma unroll
    for (int q = 0; q < QW; q++) M[q] = I[q] = D[q] = kNeg32;
    bM[w][lane] = bI[w][lane] = bD[w][lane] = kNeg32;
    __syncthreads();
    int accM = kNeg32, xJt = kNeg32;
    int xbe = fl32(fl32(mv) + entry);
    int T = -ej + 1;
    auto load = [&](int(&e)[2 * QW], int a) {
      const int *er = emit + a * (2 * Q * kWave);
#pragma unroll
      for (int q = 0; q < QW; q++) {
        e[q] = er[(q0 + q) * kWave];
        e[QW + q] = er[(Q + q0 + q) * kWave];
      }
    };
    auto row = [&](const int(&em)[2 * QW]) -> bool {
      const int wl = w > 0 ? w - 1 : W - 1;
      const int ll = w > 0 ? lane : lane - 1;
      // the value shifted into cell 0 is irrelevant: every transition into
      // it is kNeg32
      const int pM = ll >= 0 ? bM[wl][max(ll, 0)] : 0, pI = ll >= 0 ? bI[wl][max(ll, 0)] : 0,
                pD = ll >= 0 ? bD[wl][max(ll, 0)] : 0;
      // every state and table value is >= -2^30, so each add fits in int32
      // and the floors inside a maximum merge into one
#pragma unroll
      for (int q = QW - 1; q >= 0; q--) {
        const int pm = q ? M[q - 1] : pM, pi = q ? I[q - 1] : pI, pd = q ? D[q - 1] : pD;
        const int m = max(max(xbe, pm + tr[TR_MMIN][q]), max(pi + tr[TR_IMIN][q], pd + tr[TR_DMIN][q]));
        const int mn = fl32(m + em[q]);
        const int in = fl32(max(max(M[q] + tr[TR_MI][q], I[q] + tr[TR_II][q]), kNeg32) + em[QW + q]);
        accM = max(accM, mn);
        M[q] = mn;
        I[q] = in;
      }
      cM[w][lane] = M[QW - 1];
      __syncthreads();   // B1
      const int cin = ll >= 0 ? cM[wl][max(ll, 0)] : kNeg32;
      // delete chain inside the wave with minus infinity entering it
      int dc = kNeg32;
#pragma unroll
      for (int q = 0; q < QW; q++) {
        D[q] = max(fl32((q ? M[q - 1] : cin) + tr[TR_MDIN][q]), ninf_add(dc, tr[TR_DDIN][q]));
        dc = D[q];
      }
      mA[w][lane] = D[QW - 1];
      __syncthreads();   // B2
      int a = kNeg32;
#pragma unroll
      for (int j = 0; j < W; j++) a = max(mA[j][lane], ninf_add(a, bw[j]));
      // lane l-1's value (lane 0 receives 0, which is harmless: the first
      // cell's DDIN is minus infinity and every fold below starts with it)
      int cw = lane_up_i(maxplus_scan_i(a, bs));
      for (int j = 0; j < w; j++) cw = max(mA[j][lane], ninf_add(cw, bw[j]));
#pragma unroll
      for (int q = 0; q < QW; q++) D[q] = max(D[q], ninf_add(cw, pre[q]));
      // some cell reached the line that could raise xJ: its wave's maximum
      const bool trig = __builtin_amdgcn_ballot_w64(accM >= T) != 0;
      int wm = kNeg32;
      if (trig) wm = wave_max_i32(accM);
      if (lane == 0) xS[w] = wm;
      bM[w][lane] = M[QW - 1];
      bI[w][lane] = I[QW - 1];
      bD[w][lane] = D[QW - 1];
      __syncthreads();   // B3
      int m = kNeg32;
#pragma unroll
      for (int j = 0; j < W; j++) m = max(m, xS[j]);
      if (m > kNeg32) {
        xJt = max(xJt, fl32(m + ej));
        const int xB = max(fl32(mv), fl32(xJt + mv));
        xbe = fl32(xB + entry);
        T = max(xJt, 0) - ej + 1;
      }
      return false;
    };
    int ea[2 * QW], eb[2 * QW];
    int stop;
    (void)drive_rows(db.res + db.start[t], L, 0, 0, stop, lane, ea, eb, load, row);
    // the final maximum over every cell of every row, all waves (the
    // barrier first: the last row's maxima are still being read)
    {
      const int v = wave_max_i32(accM);
      __syncthreads();
      if (lane == 0) xS[w] = v;
      __syncthreads();
      int m = kNeg32;
#pragma unroll
      for (int j = 0; j < W; j++) m = max(m, xS[j]);
      if (w == 0) out.vit[uni(db.perm[t])] = fl32(fl32(m + ej) + mv);
    }
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
