// Device helpers shared by the HIP kernel files of the GPU library:
// packed 16-bit arithmetic, cross-lane moves (DPP), wave reductions and the
// row driver that streams a target's residues.  Not part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "hmm_internal.h"

namespace hmmgpu {
namespace {

typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
typedef short i16x2 __attribute__((ext_vector_type(2)));

constexpr uint32_t kNegNeg = 0x80008000u;  // two int16 -32768

__device__ __forceinline__ int uni(int v) { return __builtin_amdgcn_readfirstlane(v); }
// Saturating int32 add (one v_add_i32 with clamp): no sum can wrap.
__device__ __forceinline__ int sadd32(int a, int b) { return __builtin_elementwise_add_sat(a, b); }

// Control flow in these kernels is wave-uniform by construction, and the
// cross-lane operations (DPP, readlane, ballot, bpermute) rely on every lane
// being active.  Lane-divergent branches are therefore avoided altogether:
// per-target outputs are stored by all lanes with identical values, and the
// work counters are bumped by one lane's increment inside a wave-wide atomic.

// Wave index in the grid (scalar).
__device__ __forceinline__ int wave_id() {
  return (int)blockIdx.x * uni((int)(blockDim.x >> 6)) + (uni((int)threadIdx.x) >> 6);
}

// Wave-wide fetch-and-add of `inc` (added once per wave); returns the old
// value in a scalar.
__device__ __forceinline__ int wave_fetch_add(int32_t *p, int inc) {
  const int lane = (int)(threadIdx.x & 63);
  return uni(atomicAdd(p, lane == 0 ? inc : 0));
}

// --- packed 16-bit arithmetic ------------------------------------------------
__device__ __forceinline__ uint32_t u16_max(uint32_t a, uint32_t b) {
  return __builtin_bit_cast(uint32_t, __builtin_elementwise_max(__builtin_bit_cast(u16x2, a),
                                                                __builtin_bit_cast(u16x2, b)));
}
__device__ __forceinline__ uint32_t u16_adds(uint32_t a, uint32_t b) {
  return __builtin_bit_cast(uint32_t, __builtin_elementwise_add_sat(__builtin_bit_cast(u16x2, a),
                                                                    __builtin_bit_cast(u16x2, b)));
}
__device__ __forceinline__ uint32_t u16_subs(uint32_t a, uint32_t b) {
  return __builtin_bit_cast(uint32_t, __builtin_elementwise_sub_sat(__builtin_bit_cast(u16x2, a),
                                                                    __builtin_bit_cast(u16x2, b)));
}
__device__ __forceinline__ uint32_t i16_max(uint32_t a, uint32_t b) {
  return __builtin_bit_cast(uint32_t, __builtin_elementwise_max(__builtin_bit_cast(i16x2, a),
                                                                __builtin_bit_cast(i16x2, b)));
}
__device__ __forceinline__ uint32_t i16_adds(uint32_t a, uint32_t b) {
  return __builtin_bit_cast(uint32_t, __builtin_elementwise_add_sat(__builtin_bit_cast(i16x2, a),
                                                                    __builtin_bit_cast(i16x2, b)));
}
__device__ __forceinline__ uint32_t splat16(int v) { return ((uint32_t)(uint16_t)v) * 0x10001u; }

// --- cross-lane moves ----------------------------------------------------------
// Lane l receives lane l-1's dword (DPP wave_shr:1); lane 0 receives 0.
// A zero shifted into the first cell is harmless everywhere: every
// transition into cell 0 is minus infinity (-32768, -2^30 or probability 0),
// and adding it to 0 gives minus infinity again.
__device__ __forceinline__ uint32_t lane_up(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x138, 0xf, 0xf, true);
}
__device__ __forceinline__ int lane_up_i(int v) { return (int)lane_up((uint32_t)v); }
__device__ __forceinline__ float lane_up_f(float v) {
  return __builtin_bit_cast(float, lane_up(__builtin_bit_cast(uint32_t, v)));
}
// Packed layout: shift every 16-bit slot up by one (slot 2l <- slot 2l-1,
// slot 2l+1 <- slot 2l); slot 0 receives 0.
__device__ __forceinline__ uint32_t slot_up16(uint32_t v) {
  uint32_t prev = lane_up(v);
  return __builtin_amdgcn_alignbit(v, prev, 16);
}

__device__ __forceinline__ bool any_lane(bool p) { return __builtin_amdgcn_ballot_w64(p) != 0; }


// DPP row shift within 16-lane rows; lanes without a source get `fill`.
template <int CTRL, int ROWMASK = 0xf>
__device__ __forceinline__ float dpp_f(float v, float fill) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, fill),
                                                               __builtin_bit_cast(int, v), CTRL, ROWMASK,
                                                               0xf, false));
}
constexpr int kRowShr1 = 0x111, kRowShr2 = 0x112, kRowShr4 = 0x114, kRowShr8 = 0x118;
constexpr int kRowBcast15 = 0x142, kRowBcast31 = 0x143;

// Maximum across the wave (result uniform): an inclusive DPP max-scan of
// each 16-lane row, the rows joined by row broadcasts; lane 63 ends with the
// maximum of all 64 lanes.  No LDS round trip (a shuffle-based reduction
// costs six of them and four times the instructions).
__device__ __forceinline__ int wave_max_i32(int v) {
  constexpr int kMin = INT32_MIN;
  v = max(v, __builtin_amdgcn_update_dpp(kMin, v, kRowShr1, 0xf, 0xf, false));
  v = max(v, __builtin_amdgcn_update_dpp(kMin, v, kRowShr2, 0xf, 0xf, false));
  v = max(v, __builtin_amdgcn_update_dpp(kMin, v, kRowShr4, 0xf, 0xf, false));
  v = max(v, __builtin_amdgcn_update_dpp(kMin, v, kRowShr8, 0xf, 0xf, false));
  v = max(v, __builtin_amdgcn_update_dpp(kMin, v, kRowBcast15, 0xa, 0xf, false));
  v = max(v, __builtin_amdgcn_update_dpp(kMin, v, kRowBcast31, 0xc, 0xf, false));
  return __builtin_amdgcn_readlane(v, 63);
}

// Sum across the wave (result uniform).
__device__ __forceinline__ float wave_sum_f(float v) {
  v += dpp_f<kRowShr1, 0xf>(v, 0.0f);
  v += dpp_f<kRowShr2, 0xf>(v, 0.0f);
  v += dpp_f<kRowShr4, 0xf>(v, 0.0f);
  v += dpp_f<kRowShr8, 0xf>(v, 0.0f);
  v += dpp_f<kRowBcast15, 0xa>(v, 0.0f);
  v += dpp_f<kRowBcast31, 0xc>(v, 0.0f);
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 63));
}

// A row's lane scan as one DPP multiply-add per step (x <- x + P x_src, a
// lane without a source reading 0; rows outside the row mask keep x), and
// the wave sum's two row-broadcast steps as one DPP add each.  Each step
// states the two wait states a DPP read needs after the VALU write of its
// source.
__device__ __forceinline__ float affine_scan_fused(float a, const float (&ps)[6]) {
  asm volatile("s_nop 1\n\tv_fmac_f32_dpp %0, %0, %1 row_shr:1 row_mask:0xf bank_mask:0xf bound_ctrl:1"
               : "+v"(a) : "v"(ps[0]));
  asm volatile("s_nop 1\n\tv_fmac_f32_dpp %0, %0, %1 row_shr:2 row_mask:0xf bank_mask:0xf bound_ctrl:1"
               : "+v"(a) : "v"(ps[1]));
  asm volatile("s_nop 1\n\tv_fmac_f32_dpp %0, %0, %1 row_shr:4 row_mask:0xf bank_mask:0xf bound_ctrl:1"
               : "+v"(a) : "v"(ps[2]));
  asm volatile("s_nop 1\n\tv_fmac_f32_dpp %0, %0, %1 row_shr:8 row_mask:0xf bank_mask:0xf bound_ctrl:1"
               : "+v"(a) : "v"(ps[3]));
  asm volatile("s_nop 1\n\tv_fmac_f32_dpp %0, %0, %1 row_bcast:15 row_mask:0xa bank_mask:0xf"
               : "+v"(a) : "v"(ps[4]));
  asm volatile("s_nop 1\n\tv_fmac_f32_dpp %0, %0, %1 row_bcast:31 row_mask:0xc bank_mask:0xf"
               : "+v"(a) : "v"(ps[5]));
  return a;
}
__device__ __forceinline__ float wave_sum_fused(float v) {
  v += dpp_f<kRowShr1, 0xf>(v, 0.0f);
  v += dpp_f<kRowShr2, 0xf>(v, 0.0f);
  v += dpp_f<kRowShr4, 0xf>(v, 0.0f);
  v += dpp_f<kRowShr8, 0xf>(v, 0.0f);
  asm volatile("s_nop 1\n\tv_add_f32_dpp %0, %0, %0 row_bcast:15 row_mask:0xa bank_mask:0xf" : "+v"(v));
  asm volatile("s_nop 1\n\tv_add_f32_dpp %0, %0, %0 row_bcast:31 row_mask:0xc bank_mask:0xf" : "+v"(v));
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 63));
}

// Fused lane shifts: the previous lane's value (0 in lane 0, DPP wave_shr:1
// with bound_ctrl) enters a multiply-add or a product directly, without a
// separate move.  Each form first waits the two wait states a DPP read
// needs after the VALU write of its source.
//   acc += up(s0) t0; acc += up(s1) t1; acc += up(s2) t2   (in this order)
__device__ __forceinline__ void fmac_up3(float &acc, float s0, float t0, float s1, float t1, float s2, float t2) {
  asm volatile(
      "s_nop 1\n\t"
      "v_fmac_f32_dpp %0, %1, %2 wave_shr:1 row_mask:0xf bank_mask:0xf bound_ctrl:1\n\t"
      "v_fmac_f32_dpp %0, %3, %4 wave_shr:1 row_mask:0xf bank_mask:0xf bound_ctrl:1\n\t"
      "v_fmac_f32_dpp %0, %5, %6 wave_shr:1 row_mask:0xf bank_mask:0xf bound_ctrl:1"
      : "+v"(acc)
      : "v"(s0), "v"(t0), "v"(s1), "v"(t1), "v"(s2), "v"(t2));
}
//   up(s) t
__device__ __forceinline__ float mul_up(float s, float t) {
  float d;
  asm volatile("s_nop 1\n\tv_mul_f32_dpp %0, %1, %2 wave_shr:1 row_mask:0xf bank_mask:0xf bound_ctrl:1"
               : "=v"(d)
               : "v"(s), "v"(t));
  return d;
}

// Issue priority of a wave by the length of its target against the
// database's longest (lmax): a stage ends with its longest targets, so when
// the waves of a SIMD compete for issue, those rows go first and the
// shorter targets' waves fill the gaps.
__device__ __forceinline__ void length_priority(int L, int lmax) {
  if (4 * L > 3 * lmax)
    __builtin_amdgcn_s_setprio(3);
  else if (2 * L > lmax)
    __builtin_amdgcn_s_setprio(2);
  else if (4 * L > lmax)
    __builtin_amdgcn_s_setprio(1);
  else
    __builtin_amdgcn_s_setprio(0);
}

// Row driver.  The residues of one target arrive 256 at a time: lane j of
// `cur` holds dword j of the current 256-byte chunk, `nxt` the next chunk
// (loaded a chunk ahead).  Rows are processed four per dword with two table
// buffers in alternation: while row r is computed from one buffer, the
// table entries of row r+1 are read into the other, so memory latency is
// hidden behind a whole row of arithmetic and no buffer copy is needed.
//   load(buf, a): read the table entries of residue a into buf
//   row(buf):     compute one row from buf; return true to stop
// Rows r0 .. L-1 are run: a start inside a dword runs its first rows one at
// a time, then whole dwords (4 rows), then the last 0..3 rows one at a
// time.  With LIMIT, rows from `limit` on (a multiple of 4) are not run.
// Returns true if a row stopped the driver (`stop` = that row) or the limit
// was reached (`stop` = limit - 1).  Residue codes are valid (0..19): the
// database upload checks them.  A chunk that holds none of the target's
// rows is not fetched (its load re-reads the current chunk, already in the
// cache; no row uses the value), so reads run at most 255 bytes past a
// target, inside the database's 1 KB zero-filled tail.
// An empty use of a prefetched table buffer on a driver exit: with it the
// buffer is live on both sides of the row's stop test, so the compiler keeps
// its loads ahead of the row (otherwise they sink below the test and every
// row waits for its own table entries).
template <typename T, int N>
__device__ __forceinline__ void keep_loaded(const T (&b)[N]) {
#pragma unroll
  for (int i = 0; i < N; i++) asm volatile("" ::"v"(b[i]));
}

template <bool LIMIT = false, typename Buf, typename Load, typename Row>
__device__ __forceinline__ bool drive_rows(const uint8_t *x, int L, int r0, int limit, int &stop, int lane, Buf &ba,
                                           Buf &bb, Load load, Row row) {
  auto code = [](uint32_t w, int r) { return (int)((w >> (8 * r)) & 0xffu); };
  int r = r0;
  for (; (r & 3) != 0; r++) {
    if (r >= L) return false;
    load(ba, uni((int)x[r]));
    if (row(ba)) {
      stop = r;
      return true;
    }
  }
  if (r >= L) return false;
  const int cs = r & ~255;
  const uint32_t *p = (const uint32_t *)(x + cs);
  // chunk k of the target from cs, or chunk `own` when chunk k holds no row
  auto chunk = [&](int k, int own) { return p[(size_t)(cs + 256 * k < L ? k : own) * kWave + lane]; };
  uint32_t cur = chunk(0, 0);
  uint32_t nxt = chunk(1, 0);
  int j0 = (r & 255) >> 2;
  uint32_t w = (uint32_t)__builtin_amdgcn_readlane((int)cur, j0);
  load(ba, code(w, 0));
  for (int c0 = cs;; c0 += 256) {
    const int nfull = min(kWave, (L - c0) >> 2);  // whole dwords of rows in this chunk
    for (int j = j0; j < nfull; j++) {
      const int rr = c0 + 4 * j;
      if (LIMIT && rr >= limit) {
        stop = rr - 1;
        return true;
      }
      uint32_t wn;
      if (j == kWave - 1)
        wn = (uint32_t)__builtin_amdgcn_readlane((int)nxt, 0);
      else
        wn = (uint32_t)__builtin_amdgcn_readlane((int)cur, j + 1);
      load(bb, code(w, 1));
      if (row(ba)) {
        keep_loaded(bb);
        stop = rr;
        return true;
      }
      load(ba, code(w, 2));
      if (row(bb)) {
        keep_loaded(ba);
        stop = rr + 1;
        return true;
      }
      load(bb, code(w, 3));
      if (row(ba)) {
        keep_loaded(bb);
        stop = rr + 2;
        return true;
      }
      load(ba, code(wn, 0));
      if (row(bb)) {
        keep_loaded(ba);
        stop = rr + 3;
        return true;
      }
      w = wn;
    }
    if (nfull < kWave) {  // the target's last 0..3 rows, from dword w (row 0's table already in ba)
      const int rt = c0 + 4 * nfull;
      if (rt >= L) return false;
      if (LIMIT && rt >= limit) {
        stop = rt - 1;
        return true;
      }
      for (int k = 0; rt + k < L; k++) {
        if (k) load(ba, code(w, k));
        if (row(ba)) {
          stop = rt + k;
          return true;
        }
      }
      return false;
    }
    if (c0 + 256 >= L) return false;
    j0 = 0;
    cur = nxt;
    nxt = chunk(((c0 - cs) >> 8) + 2, ((c0 - cs) >> 8) + 1);
  }
}

__device__ __forceinline__ int sat16(int v) { return max(-32768, min(32767, v)); }
__device__ __forceinline__ int hmax16(uint32_t v) { return max((int)(int16_t)(v >> 16), (int)(int16_t)(v & 0xffffu)); }

}  // namespace
}  // namespace hmmgpu
