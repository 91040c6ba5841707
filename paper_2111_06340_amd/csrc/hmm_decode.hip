// HIP kernels (gfx950) of posterior decoding: for every selected target,
// Forward with every row kept, Backward with the posterior probability of
// each state at each residue, the target's domain regions, and one
// optimal-accuracy alignment per region (the hit's row of the multiple
// sequence alignment).
//
// One wavefront decodes one target at a time in a private scratch slot
// (one slot per resident wave; the launch has exactly one wave per slot):
//   1. Forward in fp32 probability space, as in the search's Forward
//      kernel, keeping M_k(i) and I_k(i) of every row and the row's special
//      values (N, J-loop, C-loop and E parts).
//   2. Backward from row L down to row 1.  The backward delete chain runs
//      from cell k+1 to cell k, so this phase puts virtual lane v = 63 - l
//      on physical lane l: the chain then crosses lanes in the same
//      direction as the forward one (lane l-1 -> l) and reuses its DPP
//      prefix scan.  Each row's posteriors are normalised by that row's
//      total, sum over the states that can emit residue i
//         Z_i = sum_k (fM bM + fI bI) + fN bN + fJl bJ + fCl bC,
//      which is the same value P(x) in the row's scale, so no scale factor
//      has to be tracked.  In the same pass, row by row in the same
//      direction, the region rule and the optimal-accuracy recurrence
//      (written from the end of the region, max-plus form, a 4-bit
//      traceback code per cell) advance, so posteriors are never stored.
//   3. Traceback of each region's alignment, from its start cell forwards.
// Values are kept inside [2^-32, 2^32] by exact power-of-two rescaling in
// both directions, so a product of a forward and a backward value stays far
// from the fp32 range limits.
//
// Lane-divergent branches appear only around stores (predicated writes of
// one lane's value); every cross-lane operation runs with all lanes active.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>
#include <cmath>
#include <mutex>

#include "hmm_device.h"
#include "hmm_internal.h"

// Decode scratch of hmm_decode_static: one copy per device, never freed.
// Host code must not pass this name to a kernel (on the host it is only a
// stand-in for the symbol); kernels get the address static_decode_scratch
// looked up for the current device.
static __device__ __align__(256) float scratch[hmmgpu::kStaticDecodeBytes / sizeof(float)];

namespace hmmgpu {

hipError_t static_decode_scratch(float **ptr) {
  static std::mutex mu;
  static float *addr[256] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 256) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    addr[dev] = (float *)p;
  }
  *ptr = addr[dev];
  return hipSuccess;
}

namespace {

constexpr float kNegInf = -__builtin_inff();
constexpr float kWinHi = 0x1p32f, kWinLo = 0x1p-32f;

// Lane l receives lane l-1's value; lane 0 receives `fill`.
__device__ __forceinline__ float lane_up_fill(float v, float fill) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, fill),
                                                               __builtin_bit_cast(int, v), 0x138, 0xf, 0xf, false));
}

__device__ __forceinline__ float wave_max_f(float v) {
  for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off));
  return __builtin_bit_cast(float, uni(__builtin_bit_cast(int, v)));
}

__device__ __forceinline__ int wave_min_i32(int v) {
  for (int off = 32; off >= 1; off >>= 1) v = min(v, __shfl_xor(v, off));
  return uni(v);
}

__device__ __forceinline__ float readlane_f(float v, int l) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), l));
}

// Memory written by other lanes of this wave becomes visible to its loads.
__device__ __forceinline__ void wave_fence() { __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup"); }

// Inclusive prefix scan across lanes (lane l-1 -> l) of the affine maps
// x -> a + P x, with the P parts before each step precomputed (see pstep).
__device__ __forceinline__ float affine_scan(float a, const float (&ps)[6]) {
  a = fmaf(ps[0], dpp_f<kRowShr1, 0xf>(a, 0.0f), a);
  a = fmaf(ps[1], dpp_f<kRowShr2, 0xf>(a, 0.0f), a);
  a = fmaf(ps[2], dpp_f<kRowShr4, 0xf>(a, 0.0f), a);
  a = fmaf(ps[3], dpp_f<kRowShr8, 0xf>(a, 0.0f), a);
  a = fmaf(ps[4], dpp_f<kRowBcast15, 0xa>(a, 0.0f), a);
  a = fmaf(ps[5], dpp_f<kRowBcast31, 0xc>(a, 0.0f), a);
  return a;
}
// The P parts of affine_scan for a lane's own P.
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
// The same scan in max-plus form: maps x -> max(a, x + b), b in {0, -inf}.
__device__ __forceinline__ float maxplus_scan(float a, const float (&bs)[6]) {
  a = fmaxf(a, dpp_f<kRowShr1, 0xf>(a, kNegInf) + bs[0]);
  a = fmaxf(a, dpp_f<kRowShr2, 0xf>(a, kNegInf) + bs[1]);
  a = fmaxf(a, dpp_f<kRowShr4, 0xf>(a, kNegInf) + bs[2]);
  a = fmaxf(a, dpp_f<kRowShr8, 0xf>(a, kNegInf) + bs[3]);
  a = fmaxf(a, dpp_f<kRowBcast15, 0xa>(a, kNegInf) + bs[4]);
  a = fmaxf(a, dpp_f<kRowBcast31, 0xc>(a, kNegInf) + bs[5]);
  return a;
}
__device__ __forceinline__ void maxplus_steps(float b, float (&bs)[6]) {
  bs[0] = b;
  b = b + dpp_f<kRowShr1, 0xf>(b, 0.0f);
  bs[1] = b;
  b = b + dpp_f<kRowShr2, 0xf>(b, 0.0f);
  bs[2] = b;
  b = b + dpp_f<kRowShr4, 0xf>(b, 0.0f);
  bs[3] = b;
  b = b + dpp_f<kRowShr8, 0xf>(b, 0.0f);
  bs[4] = b;
  b = b + dpp_f<kRowBcast15, 0xa>(b, 0.0f);
  bs[5] = b;
}

// Gate of a transition in the alignment recurrence: 0 if allowed, -inf if
// its probability is zero.
__device__ __forceinline__ float gate(float p) { return p > 0.0f ? 0.0f : kNegInf; }

constexpr int kDecThreads = 256;

template <int Q, bool EMIT_LDS, bool TR_LDS>
__global__ void __launch_bounds__(kDecThreads) decode_kernel(DevProfile P, DevDb db, DevDecode d) {
  extern __shared__ float ldsd[];
  constexpr int kEmit = kAlpha * 2 * Q * kWave;
  constexpr int kTr = (TR_N + 2) * Q * kWave;
  constexpr int kRowF = 2 * Q * kWave;   // floats of one stored row
  constexpr int NB = (Q + 7) / 8;        // traceback dwords per lane per row
  constexpr int kR = TR_LDS ? 1 : Q;     // register copies of a transition plane
  if (EMIT_LDS || TR_LDS) {
    if (EMIT_LDS)
      for (int i = threadIdx.x; i < kEmit / 4; i += blockDim.x) ((float4 *)ldsd)[i] = ((const float4 *)P.f_emit)[i];
    if (TR_LDS) {
      float4 *dst = (float4 *)(ldsd + (EMIT_LDS ? kEmit : 0));
      for (int i = threadIdx.x; i < kTr / 4; i += blockDim.x) dst[i] = ((const float4 *)P.f_tr)[i];
    }
    __syncthreads();
  }
  const int lane = threadIdx.x & 63;
  const int vl = 63 - lane;
  const int slot = wave_id();
  if (slot >= d.nslots) return;
  const float *emit = EMIT_LDS ? (const float *)ldsd : P.f_emit;
  const float *trp = TR_LDS ? (const float *)(ldsd + (EMIT_LDS ? kEmit : 0)) : P.f_tr;
  const int maxL = db.max_len;
  float *post = d.scratch + (size_t)slot * d.slot_dw;
  float *spec = post + (size_t)maxL * kRowF;
  int32_t *regs = (int32_t *)(spec + (size_t)maxL * 8);
  uint32_t *tbv = (uint32_t *)(regs + (size_t)maxL * 4 + 8);
  const float entry_p = P.entry_p;
  // transitions read from LDS are re-read at every use (trofs, always 0,
  // is hidden from the compiler once per row)
  int trofs = 0;
  auto trl = [&](int k, int q, int col) -> float { return trp[(k * Q + q) * kWave + col + trofs]; };

  // scan steps of the delete chains (profile constants): Forward, Backward,
  // and the alignment recurrence (max-plus form of the Backward chain)
  float psF[6], psB[6], bsB[6];
  affine_steps(trl(TR_PRE, Q - 1, lane), psF);
  affine_steps(trl(TR_SUF, 0, vl), psB);
  maxplus_steps(gate(trl(TR_SUF, 0, vl)), bsB);
  const int cbase = vl * Q;   // first cell of this lane in the Backward layout

  const int count = uni(__atomic_load_n(&db.counters[CNT_DEC], __ATOMIC_RELAXED));
  for (;;) {
    const int idx = wave_fetch_add(&db.counters[CNT_WORK_DEC], 1);
    if (idx >= count) break;
    const int t = uni(db.list_vit[idx]);
    const int L = uni(db.len[t]);
    const LenParams lp = db.lp[L];
    const float loop = lp.loop_p, move = lp.move_p;
    const uint8_t *x = db.res + db.start[t];
    const int c = uni(db.perm[t]);
    const int64_t co = db.coff[t];

    // ------------------------------------------------ 1. Forward, rows kept
    {
      float ft[TR_N + 1][kR];
      asm volatile("" : "+v"(trofs));   // per-phase table registers: no hoisting across targets
      if (!TR_LDS) {
#pragma unroll
        for (int k = 0; k <= TR_N; k++)
#pragma unroll
          for (int q = 0; q < kR; q++) ft[k][q] = trl(k, q, lane);
      }
      auto TF = [&](int k, int q) -> float { return TR_LDS ? trl(k, q, lane) : ft[k][TR_LDS ? 0 : q]; };
      float M[Q], I[Q], D[Q];
#pragma unroll
      for (int q = 0; q < Q; q++) M[q] = I[q] = D[q] = 0.0f;
      float N = 1.0f, B = move, J = 0.0f, C = 0.0f;
      int ri = 0;
      auto load = [&](float(&e)[2 * Q], int a) {
        const float *er = emit + a * (2 * Q * kWave) + lane;
#pragma unroll
        for (int q = 0; q < 2 * Q; q++) e[q] = er[q * kWave];
      };
      auto row = [&](const float(&em)[2 * Q]) -> bool {
        if (TR_LDS) asm volatile("" : "+v"(trofs));
        const float msh = lane_up_f(M[Q - 1]);
        const float ish = lane_up_f(I[Q - 1]);
        const float dsh = lane_up_f(D[Q - 1]);
        const float bent = B * entry_p;
#pragma unroll
        for (int q = Q - 1; q >= 0; q--) {
          const float pm = q ? M[q - 1] : msh, pi = q ? I[q - 1] : ish, pd = q ? D[q - 1] : dsh;
          const float sm = fmaf(pm, TF(TR_MMIN, q), fmaf(pi, TF(TR_IMIN, q), fmaf(pd, TF(TR_DMIN, q), bent)));
          const float si = fmaf(M[q], TF(TR_MI, q), I[q] * TF(TR_II, q));
          M[q] = em[q] * sm;
          I[q] = em[Q + q] * si;
        }
        const float din = lane_up_f(M[Q - 1]);
        float dc = 0.0f;
#pragma unroll
        for (int q = 0; q < Q; q++) {
          D[q] = fmaf(q ? M[q - 1] : din, TF(TR_MDIN, q), dc * TF(TR_DDIN, q));
          dc = D[q];
        }
        const float carry = lane_up_f(affine_scan(D[Q - 1], psF));
        float part = 0.0f;
#pragma unroll
        for (int q = 0; q < Q; q++) {
          D[q] = fmaf(carry, TF(TR_PRE, q), D[q]);
          part += M[q] + D[q];
        }
        float E = wave_sum_f(part);
        float Jl = J * loop, Cl = C * loop;
        J = fmaf(0.5f, E, Jl);
        C = fmaf(0.5f, E, Cl);
        N = N * loop;
        B = (N + J) * move;
        const float big = fmaxf(fmaxf(fmaxf(E, J), fmaxf(C, N)), B);
        if (big > kWinHi || big < kWinLo) {
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
          E *= s;
          Jl *= s;
          Cl *= s;
        }
        float *pr = post + (size_t)ri * kRowF + lane;
#pragma unroll
        for (int q = 0; q < Q; q++) {
          pr[q * kWave] = M[q];
          pr[(Q + q) * kWave] = I[q];
        }
        if (lane < 4) spec[ri * 8 + lane] = lane == 0 ? N : (lane == 1 ? Jl : (lane == 2 ? Cl : E));
        ri++;
        return false;
      };
      float ea[2 * Q], eb[2 * Q];
      int stop;
      (void)drive_rows(x, L, 0, 0, stop, lane, ea, eb, load, row);
    }
    wave_fence();

    // ------------------------------------------------ 2. Backward, posteriors, regions, alignments
    //
    // Rows run from L down to 1.  After row i's posteriors, the region
    // rule and the alignment recurrence advance by one row in the same
    // direction: a run of rows with core >= rt2 is a candidate region, and
    // inside it the recurrence is the optimal-accuracy one written from the
    // end of the region (T(i) = sum_{j=i}^{e} (1 - core(j))):
    //   OM_k(i) = pM_k(i) + max{ T(i+1) [end], OM_{k+1}(i+1) [MM_k],
    //                            OI_k(i+1) [MI_k], OD_{k+1}(i) [MD_k] }
    //   OI_k(i) = pI_k(i) + max{ OM_{k+1}(i+1) [IM_k], OI_k(i+1) [II_k] }
    //   OD_k(i) = max{ OM_{k+1}(i+1) [DM_k], OD_{k+1}(i) [DD_k] }
    // (a transition of probability zero is not allowed); the alignment
    // starts at the match cell maximising OM_k(i) - T(i), and its value is
    // that maximum plus T(s).  When the run ends it is kept (it held a
    // residue with core >= rt1) or its residues get code 0.
    float sum_end = 0.0f;
    int nreg = 0;
    {
      float bt[TR_N + 1][kR];   // planes 0..TR_N-1, then TR_SUF in slot TR_N
      asm volatile("" : "+v"(trofs));   // per-phase table registers: no hoisting across targets
      if (!TR_LDS) {
#pragma unroll
        for (int k = 0; k <= TR_N; k++)
#pragma unroll
          for (int q = 0; q < kR; q++) bt[k][q] = trl(k < TR_N ? k : TR_SUF, q, vl);
      }
      auto TB = [&](int k, int q) -> float {
        return TR_LDS ? trl(k, q, vl) : bt[k == TR_SUF ? TR_N : k][TR_LDS ? 0 : q];
      };
      auto GB = [&](int k, int q) -> float { return gate(TB(k, q)); };
      auto loadE = [&](float(&e)[2 * Q], int a) {
        const float *er = emit + a * (2 * Q * kWave) + vl;
#pragma unroll
        for (int q = 0; q < 2 * Q; q++) e[q] = er[q * kWave];
      };
      auto loadF = [&](float(&f)[2 * Q], int i) {   // stored row i (1-based)
        const float *pr = post + (size_t)(i - 1) * kRowF + vl;
#pragma unroll
        for (int q = 0; q < 2 * Q; q++) f[q] = pr[q * kWave];
      };
      // residues, read backwards 256 at a time (lane j holds dword j)
      uint32_t rch = 0;
      int rblk = -1;
      auto res_at = [&](int r) -> int {
        const int blk = r >> 8;
        if (blk != rblk) {
          rblk = blk;
          rch = ((const uint32_t *)(x + (size_t)blk * 256))[lane];
        }
        return (int)((((uint32_t)__builtin_amdgcn_readlane((int)rch, (r >> 2) & 63)) >> ((r & 3) * 8)) & 0xffu);
      };
      float bM[Q], bI[Q];
#pragma unroll
      for (int q = 0; q < Q; q++) bM[q] = bI[q] = 0.0f;
      float bJ = 0.0f, bN = 0.0f, bC = 0.0f;
      // alignment recurrence: row i+1 values, run state, best start cell
      float OMn[Q], OIn[Q];
#pragma unroll
      for (int q = 0; q < Q; q++) OMn[q] = OIn[q] = kNegInf;
      int in_run = 0, run_e = 0, hit = 0, besti = 0, bestc = 0;
      float T = 0.0f, nexp = 0.0f, bestv = kNegInf;
      // Rows a row ahead in two more buffers, except for long profiles,
      // where the registers are better spent on the row itself.
      constexpr bool kPrefetch = Q <= 12;
      float enx[kPrefetch ? 2 * Q : 1], fnx[kPrefetch ? 2 * Q : 1];
      float snx = 0.0f;   // special values of the next row (lanes 0..3)
      if constexpr (kPrefetch) {
#pragma unroll
        for (int q = 0; q < 2 * Q; q++) enx[q] = 0.0f;   // row L uses no emissions
        loadF(fnx, L);
        if (L >= 1) snx = spec[(L - 1) * 8 + (lane & 7)];
      }
      for (int i = L; i >= 0; i--) {
        if (TR_LDS) asm volatile("" : "+v"(trofs));
        float core = 0.0f, pend = 0.0f;
        float pm[Q], pi[Q];
        if (i >= 1) {
          // ---- Backward row i from row i+1 (ec: emissions of x_{i+1}, fc: kept Forward row i)
          const bool last = i == L;
          float ec[2 * Q], fc[2 * Q];
          float sv;
          if constexpr (kPrefetch) {
#pragma unroll
            for (int q = 0; q < 2 * Q; q++) {
              ec[q] = enx[q];
              fc[q] = fnx[q];
            }
            sv = snx;
            if (i >= 2) {
              loadE(enx, res_at(i - 1));   // residue x_i, used by row i-1
              loadF(fnx, i - 1);
              snx = spec[(i - 2) * 8 + (lane & 7)];
            }
          } else {
            if (!last) loadE(ec, res_at(i));
            loadF(fc, i);
            sv = spec[(i - 1) * 8 + (lane & 7)];
          }
          // u_k = e_k(x_{i+1}) bM_k(i+1), w_k = i_k(x_{i+1}) bI_k(i+1)
          float u[Q], w[Q];
          float part = 0.0f;
#pragma unroll
          for (int q = 0; q < Q; q++) {
            u[q] = last ? 0.0f : ec[q] * bM[q];
            w[q] = last ? 0.0f : ec[Q + q] * bI[q];
            part += u[q];
          }
          const float bB = entry_p * wave_sum_f(part);
          const float nJ = fmaf(loop, bJ, move * bB);
          const float nN = fmaf(loop, bN, move * bB);
          const float nC = last ? move : loop * bC;
          const float bE = 0.5f * (nC + nJ);
          // terms through cell k+1, formed there and moved down one cell
          float mmu[Q], imu[Q], dmu[Q];
#pragma unroll
          for (int q = 0; q < Q; q++) {
            mmu[q] = TB(TR_MMIN, q) * u[q];
            imu[q] = TB(TR_IMIN, q) * u[q];
            dmu[q] = TB(TR_DMIN, q) * u[q];
          }
          const float mm0 = lane_up_f(mmu[0]), im0 = lane_up_f(imu[0]), dm0 = lane_up_f(dmu[0]);
          // delete chain D_k = E + DM_k u_{k+1} + DD_k D_{k+1}, within the lane first
          float dp[Q];
#pragma unroll
          for (int q = Q - 1; q >= 0; q--) {
            const float dmn = q + 1 < Q ? dmu[q + 1] : dm0;
            dp[q] = q + 1 < Q ? fmaf(TB(TR_DDIN, q + 1), dp[q + 1], bE + dmn) : bE + dmn;
          }
          const float carry = lane_up_f(affine_scan(dp[0], psB));
          float mdb[Q];
#pragma unroll
          for (int q = 0; q < Q; q++) mdb[q] = TB(TR_MDIN, q) * fmaf(carry, TB(TR_SUF, q), dp[q]);
          const float md0 = lane_up_f(mdb[0]);
#pragma unroll
          for (int q = 0; q < Q; q++) {
            const float mmn = q + 1 < Q ? mmu[q + 1] : mm0;
            const float imn = q + 1 < Q ? imu[q + 1] : im0;
            const float mdn = q + 1 < Q ? mdb[q + 1] : md0;
            bM[q] = bE + mmn + fmaf(TB(TR_MI, q), w[q], mdn);
            bI[q] = fmaf(TB(TR_II, q), w[q], imn);
          }
          bJ = nJ;
          bN = nN;
          bC = nC;
          // ---- posteriors of row i, normalised by the row total
          float part2 = 0.0f;
#pragma unroll
          for (int q = 0; q < Q; q++) {
            pm[q] = fc[q] * bM[q];
            pi[q] = fc[Q + q] * bI[q];
            part2 += pm[q] + pi[q];
          }
          const float fN = readlane_f(sv, 0), fJl = readlane_f(sv, 1), fCl = readlane_f(sv, 2),
                      fE = readlane_f(sv, 3);
          const float Zc = wave_sum_f(part2);
          const float Z = fmaf(fN, bN, fmaf(fJl, bJ, fmaf(fCl, bC, Zc)));
          const float inv = 1.0f / Z;
#pragma unroll
          for (int q = 0; q < Q; q++) {
            pm[q] *= inv;
            pi[q] *= inv;
          }
          core = Zc * inv;
          pend = fE * bE * inv;
          if (d.pp && lane == 0) d.pp[co + i - 1] = core;
          sum_end += pend;
          // rescale the values carried to the next row
          const float big = fmaxf(fmaxf(fmaxf(bB, bJ), fmaxf(bN, bC)), bE);
          if (big > kWinHi || big < kWinLo) {
            int ex;
            (void)frexpf(big, &ex);
            ex = uni(ex);
            const float sc = ldexpf(1.0f, -ex);
#pragma unroll
            for (int q = 0; q < Q; q++) {
              bM[q] *= sc;
              bI[q] *= sc;
            }
            bJ *= sc;
            bN *= sc;
            bC *= sc;
          }
        }
        if (i >= 1 && core >= d.rt2) {
          // ---- one row of the alignment recurrence
          if (!in_run) {
            in_run = 1;
            run_e = i;
            hit = 0;
            T = 0.0f;
            nexp = 0.0f;
            bestv = kNegInf;
#pragma unroll
            for (int q = 0; q < Q; q++) OMn[q] = OIn[q] = kNegInf;
          }
          if (core >= d.rt1) hit = 1;
          nexp += pend;
          const float Tn = T;
          float xm[Q], xi[Q], xd[Q];
#pragma unroll
          for (int q = 0; q < Q; q++) {
            xm[q] = OMn[q] + GB(TR_MMIN, q);
            xi[q] = OMn[q] + GB(TR_IMIN, q);
            xd[q] = OMn[q] + GB(TR_DMIN, q);
          }
          const float xm0 = lane_up_fill(xm[0], kNegInf), xi0 = lane_up_fill(xi[0], kNegInf),
                      xd0 = lane_up_fill(xd[0], kNegInf);
          float dpart[Q];
#pragma unroll
          for (int q = Q - 1; q >= 0; q--) {
            const float fd = q + 1 < Q ? xd[q + 1] : xd0;
            dpart[q] = q + 1 < Q ? fmaxf(fd, dpart[q + 1] + GB(TR_DDIN, q + 1)) : fd;
          }
          const float dcar = lane_up_fill(maxplus_scan(dpart[0], bsB), kNegInf);
          float yd[Q], zd[Q];
#pragma unroll
          for (int q = 0; q < Q; q++) {
            const float od = fmaxf(dpart[q], dcar + GB(TR_SUF, q));
            yd[q] = od + GB(TR_MDIN, q);   // M_{k-1} -> D_k, formed at cell k
            zd[q] = od + GB(TR_DDIN, q);   // D_{k-1} -> D_k
          }
          const float yd0 = lane_up_fill(yd[0], kNegInf), zd0 = lane_up_fill(zd[0], kNegInf);
          uint32_t tw[NB];
#pragma unroll
          for (int j = 0; j < NB; j++) tw[j] = 0;
          T = Tn + (1.0f - core);
#pragma unroll
          for (int q = 0; q < Q; q++) {
            const float cm = q + 1 < Q ? xm[q + 1] : xm0;
            const float ci = OIn[q] + GB(TR_MI, q);
            const float cd = q + 1 < Q ? yd[q + 1] : yd0;
            float best = Tn;
            uint32_t sel = 0;
            if (cm > best) { best = cm; sel = 1; }
            if (ci > best) { best = ci; sel = 2; }
            if (cd > best) { best = cd; sel = 3; }
            const float nm = pm[q] + best;
            const float im = q + 1 < Q ? xi[q + 1] : xi0;
            const float ii = OIn[q] + GB(TR_II, q);
            const float ni = pi[q] + fmaxf(im, ii);
            const float dd = q + 1 < Q ? zd[q + 1] : zd0;
            const float dm = q + 1 < Q ? xd[q + 1] : xd0;
            tw[q >> 3] |= (sel | (ii > im ? 4u : 0u) | (dd > dm ? 8u : 0u)) << ((q & 7) * 4);
            OMn[q] = nm;
            OIn[q] = ni;
            const float v = nm - T;
            if (v > bestv && cbase + q < P.M) {
              bestv = v;
              besti = i;
              bestc = cbase + q;
            }
          }
          uint32_t *tr = tbv + (size_t)(i - 1) * NB * kWave + lane;
#pragma unroll
          for (int j = 0; j < NB; j++) tr[j * kWave] = tw[j];
        } else {
          if (in_run) {
            // the run [i+1, run_e] ends
            const int s1 = i + 1, e1 = run_e;
            if (hit) {
              const float vmax = wave_max_f(bestv);
              const int key = wave_min_i32(bestv == vmax ? (besti - 1) * (kWave * Q) + bestc : INT_MAX);
              const int32_t score = __builtin_bit_cast(int32_t, vmax + T);
              const int32_t nx = __builtin_bit_cast(int32_t, nexp);
              if (lane < 6) {
                const int32_t v = lane == 0 ? s1 : lane == 1 ? e1 : lane == 2 ? key / (kWave * Q) + 1
                                : lane == 3 ? key % (kWave * Q) : lane == 4 ? score : nx;
                regs[nreg * 8 + lane] = v;
              }
              nreg++;
            } else if (d.aln) {
              for (int j = s1 - 1 + lane; j <= e1 - 1; j += kWave) d.aln[co + j] = 0;
            }
            in_run = 0;
          }
          if (i >= 1 && d.aln && lane == 0) d.aln[co + i - 1] = 0;
        }
      }
    }
    if (d.exp_dom && lane == 0) d.exp_dom[c] = sum_end;
    wave_fence();

    // ------------------------------------------------ 3. Tracebacks of the regions
    for (int rg = 0; rg < nreg; rg++) {
      const int32_t rv = regs[rg * 8 + (lane & 7)];
      const int s1 = __builtin_amdgcn_readlane(rv, 0), e1 = __builtin_amdgcn_readlane(rv, 1);
      const int si = __builtin_amdgcn_readlane(rv, 2), sc = __builtin_amdgcn_readlane(rv, 3);
      const int32_t score = __builtin_amdgcn_readlane(rv, 4), nx = __builtin_amdgcn_readlane(rv, 5);
      // traceback codes of one diagonal, 64 cells at a time: lane j holds the
      // word of (row i0 + j, cell c0 + j); a move off that diagonal reloads
      int i0 = -(1 << 30), c0 = 0;
      uint32_t pf = 0;
      auto nib_at = [&](int i, int cc) -> uint32_t {
        int j = i - i0;
        if (!(j >= 0 && j < kWave && cc - c0 == j)) {
          i0 = i;
          c0 = cc;
          j = 0;
          const int il = min(i + lane, maxL);
          const int cl = min(cc + lane, kWave * Q - 1);
          const int vq = cl / Q, ql = cl - vq * Q;
          pf = tbv[((size_t)(il - 1) * NB + (ql >> 3)) * kWave + (63 - vq)];
        }
        const uint32_t wd = (uint32_t)__builtin_amdgcn_readlane((int)pf, j);
        return (wd >> (((cc % Q) & 7) * 4)) & 0xfu;
      };
      // codes collected 64 residues at a time, stored a window at a time
      int cw = (s1 - 1) >> 6;
      int code = 0;
      auto flush = [&](int wnd) {
        const int j = wnd * 64 + lane;
        if (d.aln && j >= s1 - 1 && j <= e1 - 1) d.aln[co + j] = (int16_t)code;
        code = 0;
      };
      auto put = [&](int r0, int v) {
        const int wnd = r0 >> 6;
        while (cw < wnd) {
          flush(cw);
          cw++;
        }
        if (lane == (r0 & 63)) code = v;
      };
      int i = si, cc = sc, st = 0;   // st: 0 = M, 2 = I, 3 = D
      int b1 = si, k2 = sc + 1;
      for (int guard = 0; guard <= (e1 - s1 + 1) + kWave * Q; guard++) {
        if (i > e1 || cc >= P.M) break;
        const uint32_t nib = nib_at(i, cc);
        if (st == 0) {
          put(i - 1, cc + 1);
          const uint32_t f = nib & 3u;
          if (f == 0) {
            b1 = i;
            k2 = cc + 1;
            break;
          }
          if (f != 3) i++;
          if (f != 2) cc++;
          st = f == 1 ? 0 : (int)f;
        } else if (st == 2) {
          put(i - 1, -(cc + 1));
          if ((nib >> 2) & 1u) {
            i++;
          } else {
            i++;
            cc++;
            st = 0;
          }
        } else {
          if ((nib >> 3) & 1u) {
            cc++;
          } else {
            i++;
            cc++;
            st = 0;
          }
        }
      }
      while (cw <= ((e1 - 1) >> 6)) {
        flush(cw);
        cw++;
      }
      const int di = wave_fetch_add(&db.counters[CNT_NDOM], 1);
      if (di < d.max_dom && lane < 9) {
        const int32_t v = lane == 0 ? c : lane == 1 ? s1 : lane == 2 ? e1 : lane == 3 ? si : lane == 4 ? b1
                        : lane == 5 ? sc + 1 : lane == 6 ? k2 : lane == 7 ? score : nx;
        ((int32_t *)(d.dom + di))[lane] = v;
      }
    }
    wave_fence();
  }
}

// Counts of the decoded alignments, one wave per domain record: every
// aligned residue for its state and residue, every step between consecutive
// states for its transition (a match-to-match step that skips nodes goes
// through their delete states).  Integer atomics, so the counts are exact.
// Records and codes are checked against the database and the profile, so
// a mismatched buffer cannot send a write out of the count table.
__global__ void __launch_bounds__(256) count_kernel(DevDb db, int M, const hmm_domain *dom, const int32_t *n_dom,
                                                    int32_t max_dom, const int16_t *aln, uint32_t *counts) {
  const int lane = threadIdx.x & 63;
  const int nw = uni((int)gridDim.x * (int)(blockDim.x >> 6));
  const int n = min(uni(*n_dom), max_dom);
  uint32_t *cm = counts, *ci = counts + (size_t)M * kAlpha, *ct = ci + (size_t)(M - 1) * kAlpha;
  enum { MM = 0, MI, MD, IM, II, DM, DD };
  for (int r = wave_id(); r < n; r += nw) {
    const int c = uni(dom[r].target);
    if (c < 0 || c >= db.n) continue;
    const int t = uni(db.iperm[c]);
    const int L = uni(db.len[t]);
    const int a1 = max(uni(dom[r].a), 1), b1 = min(uni(dom[r].b), L);
    const uint8_t *x = db.res + db.start[t];
    const int16_t *cod = aln + db.coff[t];
    for (int j = a1 - 1 + lane; j <= b1 - 1; j += kWave) {
      const int k = cod[j];
      if (k > M || k < -(M - 1) || k == 0) continue;
      const int a = x[j];
      atomicAdd(k > 0 ? &cm[(k - 1) * kAlpha + a] : &ci[(-k - 1) * kAlpha + a], 1u);
      if (j >= b1 - 1) continue;
      const int k2 = cod[j + 1];
      if (k2 > M || k2 < -(M - 1) || k2 == 0) continue;
      if (k > 0 && k2 > 0) {
        if (k2 == k + 1) {
          atomicAdd(&ct[(k - 1) * 7 + MM], 1u);
        } else if (k2 > k + 1) {
          atomicAdd(&ct[(k - 1) * 7 + MD], 1u);
          for (int kk = k + 1; kk < k2 - 1; kk++) atomicAdd(&ct[(kk - 1) * 7 + DD], 1u);
          atomicAdd(&ct[(k2 - 2) * 7 + DM], 1u);
        }
      } else if (k > 0) {
        if (-k2 == k) atomicAdd(&ct[(k - 1) * 7 + MI], 1u);
      } else if (k2 < 0) {
        if (k2 == k) atomicAdd(&ct[(-k - 1) * 7 + II], 1u);
      } else if (k2 == -k + 1) {
        atomicAdd(&ct[(-k - 1) * 7 + IM], 1u);
      }
    }
  }
}

// Targets to decode: those whose caller flags hold every bit of the mask.
__global__ void decode_select(DevDb db, const uint8_t *flags, int mask) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= db.n) return;
  const bool take = !flags || (flags[db.perm[t]] & mask) == mask;
  if (take) db.list_vit[atomicAdd(&db.counters[CNT_DEC], 1)] = (int32_t)t;
}

__global__ void decode_clear(int32_t *c) {
  if (threadIdx.x == 0) {
    c[CNT_DEC] = 0;
    c[CNT_WORK_DEC] = 0;
    c[CNT_NDOM] = 0;
  }
}

__global__ void decode_export(const int32_t *c, int32_t *n_dom) {
  if (threadIdx.x == 0) *n_dom = c[CNT_NDOM];
}

// Tables of the decode kernel: emissions in LDS up to 12 vectors per lane,
// transitions in registers up to 16, else in LDS.  (Both tables in LDS with
// workgroups of 8 waves, two waves per SIMD at 256 registers, was measured
// slower at 12 vectors: the per-row LDS reads and recomputed gates cost more
// than the second wave hides.)
template <int Q>
constexpr bool kDecEmitLds = Q <= 12;
template <int Q>
constexpr bool kDecTrLds = Q > 16;
template <int Q>
constexpr auto decode_fn = decode_kernel<Q, kDecEmitLds<Q>, kDecTrLds<Q>>;

template <int Q>
size_t decode_lds() {
  return (kDecEmitLds<Q> ? (size_t)kAlpha * 2 * Q * kWave * 4 : 0) +
         (kDecTrLds<Q> ? (size_t)(TR_N + 2) * Q * kWave * 4 : 0);
}

template <int Q>
int decode_waves_q() {
  auto k = decode_fn<Q>;
  const size_t lds = decode_lds<Q>();
  if (lds > 64 * 1024)
    (void)hipFuncSetAttribute((const void *)k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  int nb = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, k, kDecThreads, lds) != hipSuccess || nb < 1) nb = 1;
  int dev = 0, ncu = 0;
  (void)hipGetDevice(&dev);
  (void)hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev);
  if (ncu <= 0) ncu = 256;
  return nb * ncu * (kDecThreads / kWave);
}

template <int Q>
hipError_t launch_decode_q(const DevDb &db, const DevProfile &P, const DevDecode &d, hipStream_t s) {
  auto k = decode_fn<Q>;
  const size_t lds = decode_lds<Q>();
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void *)k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  // waves past the last slot return at once (after the table load)
  constexpr int wpb = kDecThreads / kWave;
  const int blocks = (d.nslots + wpb - 1) / wpb;
  hipLaunchKernelGGL(k, dim3((unsigned)blocks), dim3(kDecThreads), lds, s, P, db, d);
  return hipGetLastError();
}

#define HMM_DEC_CASES(X) \
  X(1) X(2) X(3) X(4) X(5) X(6) X(8) X(10) X(12) X(14) X(16) X(20) X(24) X(28) X(32) X(40) X(48)

}  // namespace

int decode_max_waves(const DevProfile &p) {
  switch (p.Q32) {
#define HMM_CASE(q) \
  case q:           \
    return decode_waves_q<q>();
    HMM_DEC_CASES(HMM_CASE)
#undef HMM_CASE
  }
  return 0;
}

hipError_t launch_count(const DevProfile &p, const DevDb &db, const hmm_domain *dom, const int32_t *n_dom,
                        int32_t max_dom, const int16_t *aln, uint32_t *counts, hipStream_t s) {
  const int blocks = (int)std::min<int64_t>(((int64_t)max_dom + 3) / 4, 2048);
  hipLaunchKernelGGL(count_kernel, dim3((unsigned)std::max(blocks, 1)), dim3(256), 0, s, db, p.M, dom, n_dom, max_dom,
                     aln, counts);
  return hipGetLastError();
}

hipError_t launch_decode(const DevProfile &p, const DevDb &db, const DevDecode &d, hipStream_t s) {
  hipLaunchKernelGGL(decode_clear, dim3(1), dim3(64), 0, s, db.counters);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || db.n <= 0) {
    if (e == hipSuccess) {
      hipLaunchKernelGGL(decode_export, dim3(1), dim3(64), 0, s, (const int32_t *)db.counters, d.n_dom);
      e = hipGetLastError();
    }
    return e;
  }
  const int threads = 256;
  hipLaunchKernelGGL(decode_select, dim3((unsigned)((db.n + threads - 1) / threads)), dim3(threads), 0, s, db,
                     d.sel_flags, d.sel_mask);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  switch (p.Q32) {
#define HMM_CASE(q)                          \
  case q:                                    \
    e = launch_decode_q<q>(db, p, d, s);     \
    break;
    HMM_DEC_CASES(HMM_CASE)
#undef HMM_CASE
    default:
      e = hipErrorInvalidValue;
  }
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(decode_export, dim3(1), dim3(64), 0, s, (const int32_t *)db.counters, d.n_dom);
  return hipGetLastError();
}

}  // namespace hmmgpu
