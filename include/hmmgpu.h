/*
 * hmmgpu.h -- C ABI of the MI355X (gfx950) Plan7 profile-HMM database search.
 *
 * The paper (ParaFold, arXiv 2111.06340, Background section) identifies the
 * jackhmmer searches of UniRef90 and MGnify as the CPU-bound core of
 * AlphaFold's MSA construction; its Research Motivation and Evaluation
 * sections show that CPU stage dominating end-to-end time.  The data-parallel
 * core of such a search is: score one profile HMM against every sequence of
 * a large database, through a cascade of filters.  This library runs that
 * cascade on one GPU:
 *
 *   MSV      uint8 saturating, multi-segment ungapped, on every target
 *   Viterbi  int16 saturating, gapped local, on MSV survivors
 *            (targets that saturate int16 are rescored exactly in int32)
 *   Forward  fp32 sum over all paths, on Viterbi survivors
 *
 * The model, its integer score systems and the filter cutoffs are not given
 * in the paper; the library fixes them as follows (all logs natural):
 *   - alphabet of 20 residues, codes 0..19 = A C D E F G H I K L M N P Q R S
 *     T V W Y;
 *   - match/insert scores ln(e/f), transitions ln t (t = 0 allowed);
 *   - local multihit configuration: entry ln(2/(M(M+1))) to every match
 *     state, free exit from every M and D state, E->C = E->J = ln 1/2,
 *     N/C/J loops ln(L/(L+3)), moves ln(3/(L+3));
 *   - MSV in 1/3-bit uint8 units (offset 190, per-profile bias), Viterbi in
 *     1/500-bit int16 units, both with the N/C/J loops omitted;
 *   - P-values with slope ln 2 per bit: Gumbel law for MSV and Viterbi
 *     (location mu), exponential tail for Forward (location tau).
 *
 * Conventions for every entry point:
 *   - return 0 (HMM_OK) on success, a negative HMM_E* code on failure;
 *     hmm_last_error() then holds a thread-local message;
 *   - all argument validation happens on the host before any GPU call, so a
 *     rejected call leaves no work enqueued and writes no output;
 *   - a stream argument is a hipStream_t (NULL = the default stream).
 */
#ifndef HMMGPU_H
#define HMMGPU_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define HMM_OK 0
#define HMM_EINVAL (-1)   /* bad argument: NULL pointer, M < 1, bad probabilities, bad residue code, empty sequence, offsets not increasing */
#define HMM_ERANGE (-2)   /* size beyond a library limit (M > HMM_MAX_M, sequence longer than HMM_MAX_LEN,
                             scores beyond the int32 rescore's exact range) */
#define HMM_ENOMEM (-3)   /* host or device allocation failed */
#define HMM_EDEVICE (-4)  /* a HIP runtime call failed; the message carries the HIP error string */

#define HMM_K 20          /* alphabet size */
#define HMM_MAX_M 3072    /* profile length limit: the MSV cost table must fit in LDS */
#define HMM_MAX_LEN 100000 /* target length limit */

/* Per-target flag bits written by hmm_search. */
#define HMM_MSV_PASS 0x01 /* passed the MSV filter (always set when MSV overflowed) */
#define HMM_MSV_OVF 0x02  /* MSV saturated uint8; msv = 255 */
#define HMM_VIT_RAN 0x04  /* Viterbi was computed */
#define HMM_VIT_PASS 0x08 /* passed the Viterbi filter (always set when Viterbi overflowed) */
#define HMM_VIT_OVF 0x10  /* Viterbi saturated int16; vit holds the exact int32 rescore */
#define HMM_FWD_RAN 0x20  /* Forward was computed */
#define HMM_FWD_PASS 0x40 /* Forward score passed the F3 cutoff (set for every Forward target when F3 >= 1) */
#define HMM_BIAS_PASS 0x80 /* passed the composition-bias filter (only set when the filter is on) */

typedef struct hmm_profile hmm_profile; /* opaque; library-owned; immutable after upload */
typedef struct hmm_db hmm_db;           /* opaque; library-owned; holds the packed database and search scratch */
typedef void *hmm_stream;               /* hipStream_t */

/* Probability-space profile, copied by hmm_profile_upload (fp64, row-major).
 *   bg[20]           background residue frequencies f(a)
 *   match[M][20]     match emissions of nodes 1..M
 *   insert[M-1][20]  insert emissions of nodes 1..M-1 (may be NULL when M = 1)
 *   trans[M-1][7]    MM MI MD IM II DM DD out of nodes 1..M-1 (NULL when M = 1)
 * Each emission row and bg must sum to 1 within 1e-6 with entries >= 0;
 * match entries and bg entries must be > 0 (a log-odds score must exist);
 * the MM+MI+MD, IM+II and DM+DD groups must each sum to 1 within 1e-6.
 *   mu_msv, mu_vit, tau  score-distribution locations in bits, used to turn
 *                        P-value cutoffs into score cutoffs. */
typedef struct {
  int32_t M;
  const double *bg;
  const double *match;
  const double *insert;
  const double *trans;
  double mu_msv, mu_vit, tau;
} hmm_profile_desc;

/* P-value cutoffs of the three stages; a value >= 1 passes every target.
 * bias_filter = 1 adds the composition-bias filter between MSV and Viterbi
 * (0 = off, the plain cascade): a null model with two states, one emitting
 * the background and one the profile's mean match composition
 * m(a) = (1/M) sum_k e_k(a), starting in them with probability 63/64 and
 * 1/64 and switching at each further residue with probability 1/64, gives
 * the bias score beta = ln P(x | that model) / P(x | background) (nats); a
 * target that passed MSV goes on only if MSV overflowed or
 * msv - (3/ln 2) max(beta, 0) >= the MSV cutoff of its length. */
typedef struct {
  double F1, F2, F3;
  int32_t bias_filter;
} hmm_thresholds;

/* Caller-owned DEVICE buffers of n_seqs elements each, in the caller's
 * database order.  Written asynchronously on the search stream; valid after
 * that stream synchronises.
 *   msv[i]    MSV raw score 0..255 (255 = overflow)
 *   vit[i]    Viterbi score in 1/500-bit units (exact int32 rescore after an
 *             int16 overflow); INT32_MIN when Viterbi did not run
 *   fwd[i]    Forward score in nats, raw (before the null-model correction);
 *             NaN when Forward did not run
 *   flags[i]  HMM_* flag bits
 *   counts    optional device int64[4] (may be NULL): number of MSV passes,
 *             Viterbi overflows, Viterbi passes, Forward passes
 *   bias      optional (may be NULL): the bias score beta (nats) of every
 *             MSV pass when the bias filter is on; other entries are left
 *             untouched. */
typedef struct {
  int16_t *msv;
  int32_t *vit;
  float *fwd;
  uint8_t *flags;
  int64_t *counts;
  float *bias;
} hmm_results;

/* Quantise a profile and upload its tables to the current device.  Profile
 * definition: Plan7 model as above (paper, Background section: jackhmmer's
 * profile HMM).  The descriptor's arrays are copied; they may be freed when
 * the call returns.  Blocks until the upload on `stream` completes.
 * Errors: HMM_EINVAL (NULL, M < 1, bad probabilities), HMM_ERANGE (M >
 * HMM_MAX_M), HMM_ENOMEM, HMM_EDEVICE. */
int hmm_profile_upload(const hmm_profile_desc *desc, hmm_stream stream, hmm_profile **out);

/* Release a profile (NULL is a no-op).  Must not be called while a search
 * that uses the profile is still running on the GPU. */
int hmm_profile_free(hmm_profile *p);

/* Pack and upload a sequence database (the search targets; paper,
 * Background section: the UniRef90 / MGnify sequence databases).
 *   residues   host uint8 codes 0..19, all sequences concatenated
 *   offsets    host int64[n_seqs + 1], offsets[0] = 0, strictly increasing
 *              (every sequence has length >= 1 and <= HMM_MAX_LEN)
 *   n_seqs     >= 0 (an empty database is allowed; searches then write nothing)
 * The library sorts targets by decreasing length (stable), aligns each to
 * 16 bytes on the device and keeps the permutation; results are always
 * reported in the caller's order.  Blocks until the upload completes.
 * Errors: HMM_EINVAL (NULL, bad code, bad offsets), HMM_ERANGE (too long),
 * HMM_ENOMEM, HMM_EDEVICE. */
int hmm_db_upload(const uint8_t *residues, const int64_t *offsets, int64_t n_seqs,
                  hmm_stream stream, hmm_db **out);

/* Release a database handle (NULL is a no-op); waits for its last search.
 * The packed residues are released with the last handle that uses them. */
int hmm_db_free(hmm_db *db);

/* A second handle on the same database, for concurrent searches (the paper,
 * Design section, runs the MSA searches side by side instead of one after
 * another).  The new handle shares the packed residues and index arrays of
 * `db` (no copy, no host synchronisation) and owns its own search scratch,
 * streams and events: searches on different handles are independent and
 * run concurrently when enqueued on different streams, while searches on
 * one handle stay serialised.  Free every handle with hmm_db_free, in any
 * order.  Errors: HMM_EINVAL (NULL), HMM_ENOMEM, HMM_EDEVICE. */
int hmm_db_share(const hmm_db *db, hmm_db **out);

/* Search one profile against a database: MSV on every target, Viterbi on
 * MSV survivors, int32 rescore of int16-overflowed targets, Forward on
 * Viterbi survivors.  Enqueued on `stream` without host synchronisation
 * (except when the cutoffs change, see below); allocates nothing.  The
 * search runs pipelined in chunks of the database (hmm_db_pipeline): the
 * MSV kernels run on `stream`; Viterbi and Forward of each chunk on a
 * stream owned by the database handle and the int32 rescore on another,
 * forked from `stream` and joined back before the search ends, so all of
 * the search's work is ordered on `stream`.
 * Searches on one database are serialised by the library (a search on a
 * second stream waits for the previous one on the GPU).  Changing the
 * cutoffs or the profile between searches on a database rebuilds a small
 * per-length table, which waits for the database's previous search on the
 * host.  Errors: HMM_EINVAL (NULL profile/db/thresholds/out or NULL output
 * buffer with n_seqs > 0), HMM_ERANGE (the database's longest sequence
 * times the profile's largest emission score, in the Viterbi filter's
 * 1/500-bit units, reaches 2^29: beyond that bound the int32 rescore is not
 * guaranteed exact; with a background whose rarest residue has frequency
 * 1.3 %, no emission scores above about 3,100 units, against the 5,368
 * allowed at HMM_MAX_LEN), HMM_EDEVICE. */
int hmm_search(const hmm_profile *p, hmm_db *db, const hmm_thresholds *t,
               const hmm_results *out, hmm_stream stream);

/* A group of searches of one database by n different profiles: search i is
 * profile p[i] against handle db[i] with cutoffs t[i] into out[i], and every
 * result equals that of hmm_search(p[i], db[i], &t[i], &out[i], stream).
 * The handles must be n distinct handles of one uploaded database (the
 * first from hmm_db_upload, the others from hmm_db_share).  This is the
 * many-queries mode of the paper's large-scale run (thousands of proteins,
 * each searched against the same databases; Evaluation section): the MSV
 * stage of profiles that share a kernel instance (the diagonal layout with
 * 1-3 vectors per lane, i.e. M up to 383) runs as one kernel for up to 4 of
 * them, so one wave scores a target against several profiles and the
 * residue stream and its scalar handling are shared; the other profiles'
 * MSV runs as in hmm_search.  Each search then runs its later stages on its
 * own handle's streams, concurrently with the others, all joined back into
 * `stream`.  Searches are not chunked (hmm_db_pipeline does not apply).
 * Enqueued on `stream` like hmm_search (same host waits when a handle's
 * profile or cutoffs change); allocates nothing.
 * Errors: HMM_EINVAL (n < 1; NULL array or element; a handle twice; handles
 * of different databases; bad cutoffs or NULL output buffers as in
 * hmm_search), HMM_ERANGE (as in hmm_search), HMM_EDEVICE; on an error
 * nothing is enqueued. */
int hmm_search_group(const hmm_profile *const *p, hmm_db *const *db, const hmm_thresholds *t,
                     const hmm_results *out, int32_t n, hmm_stream stream);

/* ---------------------------------------------------------------- decoding
 *
 * The step after the filter cascade: for the targets that passed it, the
 * posterior probability that each residue is emitted by the profile's core
 * (match or insert) states, the regions of each target that hold a domain,
 * and one alignment of the profile to each region -- the row that a hit
 * contributes to the multiple sequence alignment, which is what the
 * paper's MSA-construction stage (Background section) builds from its
 * jackhmmer searches.  Definitions (fp64 statements; the GPU computes in
 * fp32):
 *   - Forward and Backward over the local multihit model above give, for
 *     every residue i, P(M_k emits x_i), P(I_k emits x_i), and the core
 *     posterior core(i) = sum_k of both; end(i) = P(a domain ends at i);
 *   - a region is a maximal run of residues with core >= HMM_RT2 that
 *     holds at least one residue with core >= HMM_RT1;
 *   - in each region [s, e] the alignment is the single core path
 *     B -> M_k1 ... M_k2 -> E over residues a..b (s <= a <= b <= e; zero-
 *     probability transitions excluded) that maximises
 *       sum_{i=a}^{b} P(its state emits x_i) + sum_{i in [s,e] \ [a,b]} (1 - core(i)),
 *     the expected number of residues of the region it labels correctly. */
#define HMM_RT1 0.25f     /* a region needs one residue with core posterior >= HMM_RT1 ... */
#define HMM_RT2 0.10f     /* ... and spans a run of residues with core posterior >= HMM_RT2 */

/* One region of a decoded target and its alignment (1-based residues). */
typedef struct {
  int32_t target;   /* caller index of the target */
  int32_t s, e;     /* region: residues s..e */
  int32_t a, b;     /* aligned residues a..b */
  int32_t k1, k2;   /* first and last match node of the alignment */
  float score;      /* the maximised objective above */
  float nexp;       /* expected number of domain ends inside the region: sum of end(i), i = s..e */
} hmm_domain;

/* Caller-owned DEVICE outputs of hmm_decode.
 *   dom       [max_dom] domain records, in no particular order
 *   n_dom     int32[1]: number of regions found (records beyond max_dom are
 *             counted but not written)
 *   exp_dom   [n_seqs] caller order, or NULL: expected number of domains
 *             (sum of end(i) over the target) of each decoded target;
 *             other entries are left untouched
 *   pp        [n_residues] float, laid out like the caller's residue
 *             array, or NULL: core(i) of every residue of a decoded target
 *   aln       [n_residues] int16, laid out like the caller's residue array,
 *             or NULL: for every residue of a decoded target, +k if its
 *             region's alignment puts it on M_k, -k on I_k, 0 otherwise. */
typedef struct {
  hmm_domain *dom;
  int32_t max_dom;
  int32_t *n_dom;
  float *exp_dom;
  float *pp;
  int16_t *aln;
} hmm_decode_out;

/* Posterior decoding, domain regions and alignments of the targets whose
 * flags (device uint8[n_seqs], caller order; e.g. the flags a search wrote)
 * contain every bit of `mask`; flags = NULL decodes every target.  The
 * profile must be the one the flags came from.  Enqueued on `stream`;
 * serialised with the searches on `db`.  On its first call for a database
 * (and when a longer profile needs more) the library allocates a scratch
 * area on the device for the Forward/Backward matrices of the targets in
 * flight -- one slot per resident wave, at most 16 GiB -- which the
 * database keeps until hmm_db_free.  Errors: HMM_EINVAL (NULL profile, db
 * or out; NULL dom or n_dom; max_dom < 0), HMM_ENOMEM (scratch),
 * HMM_EDEVICE. */
int hmm_decode(const hmm_profile *p, hmm_db *db, const uint8_t *flags, uint8_t mask,
               const hmm_decode_out *out, hmm_stream stream);

/* hmm_decode for callers that cannot allocate device memory: code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc.  The
 * arguments, outputs and results are hmm_decode's; the per-wave scratch is
 * a fixed array of 512 MiB that the library holds on every device it runs
 * on (one copy per device, from the first call on that device until the
 * process ends), so the call allocates nothing.  Slots are sized for the
 * database's longest target; as many waves run as slots fit (a multiple of
 * four): M = 734 with targets up to 1,000 residues gives 80 waves, M = 2,500
 * with targets up to 5,000 residues 4.  Every call on one device shares
 * the array and keeps no state in it between calls (nothing in it needs to
 * start at zero), so calls that overlap on one device -- on different
 * streams, or from different threads -- race and give undefined results;
 * calls serialised on one stream are safe.  Errors: those of hmm_decode
 * (HMM_ENOMEM aside), and HMM_ERANGE when four slots exceed the array. */
int hmm_decode_static(const hmm_profile *p, hmm_db *db, const uint8_t *flags, uint8_t mask,
                      const hmm_decode_out *out, hmm_stream stream);

/* ---------------------------------------------------------------- iteration
 *
 * A jackhmmer search is iterated: the hits it accepts are aligned to the
 * profile and a new profile is estimated from that alignment for the next
 * search (the paper, Background section, names jackhmmer as the search tool
 * of the MSA stage).  Counting runs on the GPU; the estimate is a small
 * host computation:
 *   - every aligned residue counts once for its state (M_k or I_k) and
 *     residue; every step between consecutive states of an alignment's path
 *     counts once for its transition, where M_k -> M_k' (k' > k + 1) passes
 *     through D_{k+1} .. D_{k'-1} (MD_k, DD_{k+1} .. DD_{k'-2}, DM_{k'-1});
 *   - the new profile takes the old one as a Dirichlet prior:
 *       e'_k(a) = (c_k(a) + A e_k(a)) / (sum_b c_k(b) + A)   (match and insert rows)
 *       t'_k    = (n_k + B t_k) / (sum of the group's n + B)  (MM MI MD | IM II | DM DD). */

/* Add the counts of the alignments of dom[0 .. min(*n_dom, max_dom)) to
 * `counts` (device uint32 [M][20] match, then [M-1][20] insert, then
 * [M-1][7] transitions MM MI MD IM II DM DD; not cleared here).  dom, n_dom
 * and aln are hmm_decode's outputs (device), on the same database and
 * profile.  Enqueued on `stream` after the database's previous work.
 * Errors: HMM_EINVAL (NULL argument, max_dom < 0), HMM_EDEVICE. */
int hmm_count(const hmm_profile *p, hmm_db *db, const hmm_domain *dom, const int32_t *n_dom, int32_t max_dom,
              const int16_t *aln, uint32_t *counts, hmm_stream stream);

/* Host: the next iteration's probability profile from host counts (layout
 * as hmm_count's) and the prior profile, with prior weights A (emissions)
 * and B (transitions) > 0.  Writes match[M][20], insert[M-1][20],
 * trans[M-1][7] (caller-owned, fp64).  Errors: HMM_EINVAL (invalid prior,
 * NULL, A or B not > 0). */
int hmm_rebuild(const hmm_profile_desc *prior, const uint32_t *counts, double A, double B, double *match,
                double *insert, double *trans);

/* Profiling hook: record HIP events around each stage of the next searches
 * on this database, in a ring of `capacity` searches (0 turns it off).  The
 * events are recorded on the search stream, so they bracket exactly that
 * stream's kernels.  Errors: HMM_EINVAL (NULL db, capacity < 0),
 * HMM_EDEVICE. */
int hmm_db_stage_timing(hmm_db *db, int32_t capacity);

/* Stage durations (ms) of the recorded searches, oldest first:
 * out_ms[4*i + s] for search i and stage s = MSV, Viterbi int16, int32
 * rescore, Forward (each including its small list/counter kernels).  The
 * rescore and Forward run concurrently (the rescore on a stream internal to
 * the database, forked from and joined back into the search stream): both
 * are timed from the end of the int16 Viterbi stage, the rescore to its own
 * end and Forward to the end of both, so Forward's figure is the time the
 * two together add to the search.  When the three stages after MSV run as
 * one kernel (hmm_db_fused_tail), the Viterbi figure holds all three.  At most `cap` searches are returned,
 * their number in *n.  Waits for the recorded searches to finish and
 * clears the record.  Errors: HMM_EINVAL, HMM_EDEVICE. */
int hmm_db_stage_times(hmm_db *db, float *out_ms, int32_t cap, int32_t *n);

/* Measurement hook: the packed 16-bit VALU rate this device sustains, in
 * element-ops per second (one wave64 packed instruction = 128), from a timed
 * kernel of independent chains of the MSV recurrence's two instructions
 * (packed fp16 add and maximum) at 32 waves per CU: the practical ceiling of
 * the integer filters, beside the datasheet peak 256 CU x 64 lanes x 2 x
 * 2.4 GHz = 78.64e12.  Allocates and frees a work buffer of 4 bytes per
 * thread of the launch (2 MB on 256 CUs); synchronises `stream`.  *ms
 * (if non-NULL) receives the timed launch's duration.
 * Errors: HMM_EINVAL (NULL ops_per_s), HMM_ENOMEM, HMM_EDEVICE. */
int hmm_probe_pk16(hmm_stream stream, double *ops_per_s, float *ms);

/* Tuning hook: the number of chunks (1..8) a search on this handle is
 * pipelined in.  The length-sorted targets are split into that many
 * contiguous ranges of about equal residue counts; the MSV kernels of the
 * chunks run back to back on the search stream while the Viterbi, rescore
 * and Forward of each finished chunk run on the handle's own streams beside
 * them.  Results do not depend on it.  chunks = 0 changes nothing;
 * *current (if non-NULL) receives the count in force.  The default is 1
 * (plain sequential stages, which is also what per-stage timing needs).
 * Errors: HMM_EINVAL (NULL db, chunks outside 0..8). */
int hmm_db_pipeline(hmm_db *db, int32_t chunks, int32_t *current);

/* Tuning hook: how a search on this handle runs the stages after MSV.
 * mode 1: one kernel per stage (int16 Viterbi over every MSV survivor, then
 * the int32 rescore of its overflows beside Forward over its passes).
 * mode 2: for profiles of at most 384 nodes, one kernel in which a wave
 * takes each MSV survivor through its Viterbi, rescore (if it overflowed)
 * and Forward (if it passed) before its next target, so that no stage
 * waits for the longest target of the one before it; longer profiles run
 * the staged kernels.  mode 3 (the default): mode 2 for searches whose
 * Viterbi cutoff F2 is 1 (every target that reaches Viterbi reaches
 * Forward), mode 1 otherwise.  Results do not depend on it.  When the fused
 * kernel runs, hmm_db_stage_times reports it as the Viterbi stage.  mode 0
 * changes nothing; *current (if non-NULL) receives the mode in force.
 * Errors: HMM_EINVAL (NULL db, mode outside 0..3). */
int hmm_db_fused_tail(hmm_db *db, int32_t mode, int32_t *current);

/* Database properties: number of targets, total residues, longest target. */
int hmm_db_info(const hmm_db *db, int64_t *n_seqs, int64_t *n_residues, int32_t *max_len);

/* Human-readable text of a status code (static storage). */
const char *hmm_strerror(int status);

/* Message of the last failed call on this thread ("" if none). */
const char *hmm_last_error(void);

/* Test hook: quantise a profile descriptor on the host exactly as
 * hmm_profile_upload does, without touching the GPU.
 *   scalars   int32[8]: BIAS8, ENTRY8, EXIT8, ENTRY16, EJ16, M, Q8, Q32
 *             (Q8 / Q32: vectors per lane of the 16-bit / 32-bit layouts)
 *   cost8     uint8[M][20]   MSV costs (may be NULL)
 *   msc16     int16[M][20]   Viterbi match scores (may be NULL)
 *   isc16     int16[M-1][20] Viterbi insert scores (may be NULL)
 *   t16       int16[M-1][7]  Viterbi transitions (may be NULL)
 * Errors: as hmm_profile_upload's validation (HMM_EINVAL, HMM_ERANGE). */
int hmm_debug_tables(const hmm_profile_desc *desc, int32_t *scalars, uint8_t *cost8,
                     int16_t *msc16, int16_t *isc16, int16_t *t16);

/* Test hook: the per-length parameters a search uses for target length L
 * under cutoffs t (host computation, no GPU call).
 *   i32[6]: MOVE8, THR8, MOVE16, THR16, 0, 0
 *   f64[4]: LOOP, MOVE (nats), NULL(L) (nats), Forward cutoff (nats; -inf
 *           when F3 >= 1)
 * Errors: HMM_EINVAL (NULL argument, L < 1, invalid descriptor). */
int hmm_debug_length_params(const hmm_profile_desc *desc, const hmm_thresholds *t, int32_t L,
                            int32_t *i32, double *f64);

#ifdef __cplusplus
}
#endif

#endif /* HMMGPU_H */
