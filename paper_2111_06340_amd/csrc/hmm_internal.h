// Internal declarations shared by the host side (hmm_host.cpp) and the
// kernels (hmm_kernels.hip) of the GPU library.  Not part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "hmmgpu.h"

namespace hmmgpu {

constexpr int kWave = 64;           // CDNA wavefront
constexpr int kAlpha = 20;          // residue alphabet
constexpr int kBase8 = 190;         // MSV offset of the N/J start
constexpr int kNeg16 = -32768;      // int16 "minus infinity"
constexpr int32_t kNeg32 = -(1 << 30);  // int32 rescore floor
constexpr int kMaxQ8 = 24;          // 128 cells per packed vector -> M <= 3072
constexpr int kMaxQDiag = 14;       // largest MSV diagonal-layout instance (LDS 10 KB per vector)
constexpr int kMaxQ32 = 48;         // 64 cells per 32-bit vector -> M <= 3072

// Transition planes of the per-cell "into" layout (cell k = node k+1).
//   MMIN/IMIN/DMIN: M_k, I_k, D_k (node k) -> M_{k+1};  MDIN/DDIN: M_k, D_k
//   -> D_{k+1};  MI/II: M_{k+1}/I_{k+1} -> I_{k+1}.  Structural and padding
//   cells hold the type's minus infinity (probability 0 in Forward).
enum { TR_MMIN = 0, TR_IMIN, TR_DMIN, TR_MDIN, TR_DDIN, TR_MI, TR_II, TR_N };

// Per-target-length parameters, one entry per L = 0..max_len.
struct LenParams {
  int32_t move8;    // MSV cost of N->B / J->B / C->T
  int32_t thr8;     // MSV pass: msv_raw >= thr8 (0..256)
  int32_t move16;   // Viterbi score of the moves (<= 0)
  int32_t thr16;    // Viterbi pass: vit >= thr16
  float loop_p;     // Forward N/C/J self-loop probability L/(L+3)
  float move_p;     // Forward move probability 3/(L+3)
  float fthr;       // Forward pass: fwd > fthr (nats); -inf when F3 >= 1
  float pad;
};

// Device-side profile, passed to kernels by value.
struct DevProfile {
  int32_t M, Q8, Q32;
  int32_t Qm;                   // vectors per lane of the MSV kernel
  int32_t msv_diag;             // MSV layout: 1 diagonal, 0 striped (see msv below)
  int32_t bias8, entry8, exit8;
  int32_t entry16, ej16;
  // Largest D->M transition score over the nodes (int16 and int32 scales;
  // minus infinity when M = 1): a delete value d with d + dm_max <= the
  // B->M entry value can no longer change any match cell.
  int32_t dm_max16, dm_max32;
  float entry_p;                // 2/(M(M+1))
  float bias_r[kAlpha];         // composition-bias filter: mean match emission / background
  // MSV table, packed fp16 scores E = BIAS8 - COST8 (padding cells -1024).
  // msv_diag = 1: [20][P], P = 128 Qm, dword c = (E_c, E_{(c + P/2) mod P});
  // msv_diag = 0: [20][Qm][64] in the striped packed layout.
  const uint32_t *msv;
  const uint32_t *vit_emit;     // [20][2][Q8][64] packed i16: msc plane, isc plane
  const uint32_t *vit_tr;       // [TR_N][Q8][64] packed i16
  const int32_t *v32_emit;      // [20][2][Q32][64]
  const int32_t *v32_tr;        // [TR_N][Q32][64]
  const float *f_emit;          // [20][2][Q32][64] odds e/f, i/f
  // [TR_N + 3][Q32][64]: probabilities; plane TR_PRE: D-chain products
  // prod_{j<=q} DDIN(lane*Q + j); plane TR_SUF: prod_{j=q+1}^{Q} DDIN(lane*Q + j)
  // (the last factor belongs to the next lane's first cell; 0 past the end);
  // plane TR_EXIT: exit weight g_c of cell c (see hmm_profile_upload), so
  // that a row's E = sum_c M_c g_c
  const float *f_tr;
};
enum { TR_PRE = TR_N, TR_SUF = TR_N + 1, TR_EXIT = TR_N + 2 };

// Counters in the database scratch (device int32).
enum {
  CNT_VIT = 0, CNT_OVF, CNT_FWD, CNT_FWD_PASS, CNT_WORK_VIT, CNT_WORK_OVF, CNT_WORK_FWD,
  CNT_DEC, CNT_WORK_DEC, CNT_NDOM,   // posterior decoding: list size, work counter, domains found
  CNT_WORK_MSV,                      // MSV: runs of targets taken
  CNT_N = 16
};

struct DevDb {
  int64_t n;
  int32_t max_len;
  const uint8_t *res;           // packed residues, each target 16-byte aligned
  const int64_t *start;         // [n] byte offset of each target (sorted order)
  const int32_t *len;           // [n]
  const int32_t *perm;          // [n] sorted index -> caller index
  uint8_t *flags_sorted;        // [n] scratch: every stage's flags, sorted order
  int16_t *msv_sorted;          // [n] scratch: MSV scores, sorted order
  int32_t *list_vit;            // [n] MSV survivors (sorted indices)
  int32_t *list_ovf;            // [n] int16 Viterbi overflows
  int32_t *list_fwd;            // [n] Viterbi survivors
  int32_t *counters;            // [CNT_N]
  const LenParams *lp;          // [max_len + 1]
  const int64_t *coff;          // [n] offset of each target in the caller's residue array
  const int32_t *iperm;         // [n] caller index -> sorted index
  int32_t prio_by_len;          // 1: the later stages' waves take issue priority by target length
};

struct DevOut {
  int16_t *msv;
  int32_t *vit;
  float *fwd;
  uint8_t *flags;
  int64_t *counts;
  float *bias;                  // optional bias scores
  int32_t bias_filter;          // 1: composition-bias filter between MSV and Viterbi
  int32_t fused_tail;           // 1: the stages after MSV as one kernel where an instance exists
};

// Posterior decoding (hmm_decode): outputs and per-wave scratch.
struct DevDecode {
  hmm_domain *dom;              // [max_dom] domain records
  int32_t max_dom;
  int32_t *n_dom;               // device int32: domains found (may exceed max_dom)
  float *exp_dom;               // [n] caller order, or null
  float *pp;                    // [n_residues] caller layout, or null
  int16_t *aln;                 // [n_residues] caller layout, or null
  const uint8_t *sel_flags;     // [n] caller order; null = decode every target
  int32_t sel_mask;             // decode targets with (flags & mask) == mask
  float rt1, rt2;               // region thresholds on the core posterior
  float *scratch;               // nslots * slot_dw floats
  int64_t slot_dw;              // dwords per wave slot
  int32_t nslots;               // waves of the decode launch (one slot each)
};

// Dwords of one decode slot for vectors-per-lane Q and targets up to max_len:
//   kept Forward rows [max_len][2][Q][64], their specials [max_len][8],
//   regions [max_len / 2 + 1][8], traceback codes [max_len][ceil(Q/8)][64].
inline int64_t decode_slot_dw(int Q, int max_len) {
  const int64_t nb = (Q + 7) / 8;
  const int64_t dw = (int64_t)max_len * (2 * Q * 64 + 8 + 4 + nb * 64) + 8;
  return (dw + 63) / 64 * 64;
}

// Largest number of waves of the decode kernel of profile p resident at once.
int decode_max_waves(const DevProfile &p);

// Enqueue the decode of the selected targets on `stream` (d.nslots waves).
hipError_t launch_decode(const DevProfile &p, const DevDb &db, const DevDecode &d, hipStream_t stream);

// Bytes of the decode scratch held in a file-scope device array, for the
// entry point that allocates nothing (hmm_decode_static).
constexpr size_t kStaticDecodeBytes = (size_t)512 << 20;

// Device address of that array on the current device: looked up once per
// device (hipGetSymbolAddress) and kept for the life of the process.
hipError_t static_decode_scratch(float **ptr);

// Forward and int32 rescore of long profiles with one workgroup of several
// waves per target (hmm_coop.hip): coop_instance(Q) tells whether vectors
// per lane Q have such an instance.
bool coop_instance(int Q);
hipError_t launch_fwd_coop(const DevProfile &p, const DevDb &db, const DevOut &o, hipStream_t stream);
hipError_t launch_vit32_coop(const DevProfile &p, const DevDb &db, const DevOut &o, hipStream_t stream);

// A search runs in up to kMaxChunks chunks of the length-sorted database
// (contiguous ranges of about equal residue counts), pipelined: the MSV
// kernels of the chunks run back to back on the search stream, and the rest
// of each chunk's cascade (Viterbi, then Forward, with the int32 rescore
// beside it) on a second stream as soon as the chunk's MSV is done, so it
// overlaps the next chunk's MSV.  Each chunk has its own counter block and
// keeps its survivor lists inside its own index range.
constexpr int kMaxChunks = 8;

// Streams and events that order one database handle's searches.
struct SearchSync {
  hipStream_t tail = nullptr;           // Viterbi and Forward of the chunks
  hipStream_t aux = nullptr;            // int32 rescore, beside Forward
  hipEvent_t msv_done[kMaxChunks] = {}; // recorded on the search stream
  hipEvent_t vit_done[kMaxChunks] = {}; // recorded on tail
  hipEvent_t aux_done = nullptr, tail_done = nullptr;
};

// The sorted targets [a, b) as a database of their own, with counter block k.
inline DevDb chunk_of(const DevDb &d, int64_t a, int64_t b, int k) {
  DevDb c = d;
  c.n = b - a;
  c.start += a;
  c.len += a;
  c.perm += a;
  c.coff += a;
  c.flags_sorted += a;
  c.msv_sorted += a;
  c.list_vit += a;
  c.list_ovf += a;
  c.list_fwd += a;
  c.counters += (size_t)k * CNT_N;
  return c;
}

// Enqueue the whole cascade of the chunks chunk[0..nchunks) on `stream`;
// all of its work is joined back into `stream` before the final counter
// export (the sum over the chunks' counter blocks, which start at
// chunk[0].counters).  When `ev` is non-null, ev[0..4] are recorded at the
// start and after the last MSV (search stream), after the last Viterbi
// (tail), after the last rescore (aux) and at the end (search stream).
hipError_t launch_search(const DevProfile &p, const DevDb *chunk, int nchunks, const DevOut &out,
                         hipStream_t stream, const SearchSync &sync, hipEvent_t *ev);

// Enqueue a group of n one-chunk searches of one database (one handle each):
// MSV of profiles sharing a diagonal instance as group kernels, then each
// search's tail on its own streams y[i], joined back into `stream`.
hipError_t launch_search_group(const DevProfile *P, const DevDb *db, const DevOut *o, int n, hipStream_t stream,
                               const SearchSync *const *y);

// Enqueue the emission and transition counts of the alignments of
// dom[0 .. min(*n_dom, max_dom)) (codes in aln, caller residue layout) into
// counts: uint32 [M][20] match, [M-1][20] insert, [M-1][7] transitions.
hipError_t launch_count(const DevProfile &p, const DevDb &db, const hmm_domain *dom, const int32_t *n_dom,
                        int32_t max_dom, const int16_t *aln, uint32_t *counts, hipStream_t stream);

// The packed 16-bit VALU rate the device sustains (element-ops per second),
// measured by a timed kernel of independent add/maximum chains; scratch
// holds one word per thread of the launch (2 x CUs x 1024).
hipError_t probe_pk16(uint32_t *scratch, int64_t scratch_words, hipStream_t stream, double *ops_per_s,
                      float *ms);

// Number of packed vectors per lane.
inline int q8_of(int M) { return (M + 2 * kWave - 1) / (2 * kWave); }
inline int q32_of(int M) { return (M + kWave - 1) / kWave; }

}  // namespace hmmgpu
