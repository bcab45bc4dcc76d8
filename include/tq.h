/*
 * tq.h -- C ABI of the TurboQuant search hot path for AMD Instinct MI355X
 * (gfx950), as studied in "TurboVec" (arXiv 2607.16973).
 *
 * The library compresses L2-normalisable float32 embeddings with TurboQuant
 * (section II-B: normalise, rotate with one seeded orthogonal matrix,
 * Lloyd-Max scalar quantisation against boundaries derived analytically from
 * the post-rotation coordinate law, bit packing, length-renormalised scoring)
 * and answers brute-force top-k inner-product queries over the codes, with
 * kernel-level multi-tenant allowlist filtering (section III-B).
 *
 * Conventions for every entry point
 * ---------------------------------
 *  - Pointers named *_dev are device (HBM) pointers on the current HIP device;
 *    pointers named *_host are host pointers.  The caller owns every pointer
 *    argument; the library never keeps one after the call returns.  The
 *    library owns only the opaque handles and the storage inside them.
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *    Device work is enqueued on it and is asynchronous: outputs are valid
 *    once the stream has been synchronised, and inputs must stay alive and
 *    unmodified until then.
 *  - Every function returns a tq_status and never throws or aborts.
 *    Arguments are validated before any device work is enqueued; on error
 *    nothing is enqueued and tq_last_error() describes the failure.
 *  - Functions that need a GPU return TQ_EDEVICE when none is usable.  The
 *    codebook and rotation constructors are host-only and work without one.
 *  - Sizes: 64 <= d <= 2048 with d % 64 == 0; bits in {1, 2, 3, 4, 8}
 *    (bits == 3 additionally needs d % 128 == 0); k in 1..4096.
 *  - Environment: TQ_SCAN_GRID=<n> (1..65535) sets the number of workgroups
 *    of the search kernels, read at each call (default: one per compute
 *    unit; other values are ignored).  Results do not depend on it; it
 *    exists to test large per-workgroup shares of the index at small sizes.
 */
#ifndef TQ_H
#define TQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    TQ_OK = 0,
    TQ_EINVAL = -1,          /* bad argument (null pointer, bad size, bad id) */
    TQ_ENOMEM = -2,          /* device or host allocation failed */
    TQ_EDEVICE = -3,         /* no usable GPU, or a HIP runtime error */
    TQ_EUNSUPPORTED = -4     /* valid request outside what the library supports */
} tq_status;

typedef struct tq_codebook tq_codebook;
typedef struct tq_rotation tq_rotation;
typedef struct tq_index tq_index;

/* Message for the last failed call on this thread (static storage, never
 * NULL; "" if none). */
const char *tq_last_error(void);

/* Library version string, e.g. "tq 0.1.0 gfx950". */
const char *tq_version(void);

/* ------------------------------------------------------------- codebook ----
 * build_codebook(d, b) -- section II-B step 3.  Lloyd-Max scalar quantiser
 * with L = 2^bits levels for the law of one coordinate of a uniformly random
 * unit vector in R^d (density proportional to (1 - x^2)^((d-3)/2), the
 * paper's "Beta / N(0, 1/d)" marginal).  No data is involved: the tables
 * depend on (d, bits) only.  Host-only, float64, deterministic.
 * Errors: TQ_EINVAL for d out of range, TQ_EUNSUPPORTED for other bits,
 * TQ_EINVAL for out == NULL. */
tq_status tq_build_codebook(int32_t d, int32_t bits, tq_codebook **out);

/* Copies the float64 tables: bounds_host[L-1] (strictly increasing, the
 * middle one exactly 0) and cents_host[L] (strictly increasing,
 * antisymmetric).  Either pointer may be NULL to skip it. */
tq_status tq_codebook_tables(const tq_codebook *cb, double *bounds_host,
                             double *cents_host);

/* Per-coordinate distortion E[(X - Q(X))^2] of the codebook (float64). */
tq_status tq_codebook_mse(const tq_codebook *cb, double *mse_out);

void tq_codebook_free(tq_codebook *cb);

/* ------------------------------------------------------------- rotation ----
 * Rotation R(seed) -- section II-B step 2 (one orthogonal matrix, drawn
 * at random once and then fixed).  Haar-distributed d x d orthogonal matrix: a d x d matrix of
 * standard normals (SplitMix64 counter stream of `seed`, 53-bit uniforms,
 * Box-Muller on consecutive pairs, row-major) factored by Householder QR,
 * with columns sign-corrected so the triangular factor has a positive
 * diagonal; stored as float32 row-major.  y = R x, i.e. y_j = sum_k R[j][k]
 * x_k.  Host-only (the device copy is made on first device use).
 * Errors: TQ_EINVAL for d out of range or out == NULL. */
tq_status tq_rotation_create(int32_t d, uint64_t seed, tq_rotation **out);

/* Copies the float32 matrix, row-major, d*d floats, to R_host. */
tq_status tq_rotation_matrix(const tq_rotation *rot, float *R_host);

void tq_rotation_free(tq_rotation *rot);

/* --------------------------------------------------------------- encode ----
 * rotate_quantize(X) -> codes + scales -- section II-B steps 1-5.
 * For each float32 row x of X_dev [n][d] (row-major):
 *   n_x    = ||x|| (float64);
 *   code_j = number of boundaries t_i with fl64(t_i * n_x) <= (R x)_j, where
 *            (R x)_j is the float64 sum over k = 0..d-1 in order (a value on
 *            a boundary goes to the upper cell; a zero row codes to L/2);
 *   scale  = n_x / ||c[code]|| (float64, stored float32): the per-vector
 *            length-renormalisation scalar; 0 for a zero row.
 * The rotation runs on the matrix cores (float32 MFMA with float64
 * accumulation); coordinates whose MFMA value lies within a proven error
 * bound of a boundary are recomputed exactly, so the codes equal the
 * definition above bit for bit.
 * Outputs: codes_dev [n][d*bits/8] bytes in the canonical layout (one
 * little-endian bitstream per row, coordinate j at bits [bits*j, bits*j +
 * bits), least significant bit first); scales_dev [n] float32.
 * Errors: TQ_EINVAL for a null pointer, n < 0, or mismatched (d, bits)
 * between cb and rot; a non-finite input value makes the call return
 * TQ_EINVAL after synchronising `stream` (the outputs are then unspecified). */
tq_status tq_rotate_quantize(const tq_codebook *cb, const tq_rotation *rot,
                             const float *X_dev, int64_t n, uint8_t *codes_dev,
                             float *scales_dev, void *stream);

/* ------------------------------------------------------- query rotation ----
 * q' = R q for every row of Q_dev [nq][d] float32 -> Qrot_dev [nq][d]
 * float32 (section II-B step 2 applied to queries; queries are not
 * normalised).  Exposed so the query rotation can be checked on its own;
 * tq_search performs it internally. */
tq_status tq_rotate_queries(const tq_rotation *rot, const float *Q_dev,
                            int64_t nq, float *Qrot_dev, void *stream);

/* ------------------------------------------------------------ index -------
 * TurboQuantIndex (section III-A): flat scan, positional ids (the i-th
 * vector added has id i), online ingest with no training.  n_tenants in
 * 1..65535 sets the allowlist width W = ceil(n_tenants / 64) words.  The
 * codebook and rotation are copied; the caller may free them afterwards. */
tq_status tq_index_create(const tq_codebook *cb, const tq_rotation *rot,
                          int32_t n_tenants, tq_index **out);

/* Pre-allocates device storage for `capacity` vectors and uploads the
 * index's rotation matrix to the current device (a one-time set-up that the
 * first add would otherwise do). */
tq_status tq_index_reserve(tq_index *idx, int64_t capacity);

/* add(): encodes X_dev [n][d] float32 exactly as tq_rotate_quantize and
 * appends the vectors, with tenant ids tenants_dev [n] uint16 (NULL = tenant
 * 0 for all).  A tenant id >= n_tenants is reported as TQ_EINVAL after
 * synchronising `stream` (the vectors are then not added). */
tq_status tq_index_add(tq_index *idx, const float *X_dev,
                       const uint16_t *tenants_dev, int64_t n, void *stream);

/* Appends vectors given as canonical codes_dev [n][d*bits/8] and scales_dev
 * [n] float32 (as produced by tq_rotate_quantize), with tenants as above. */
tq_status tq_index_add_codes(tq_index *idx, const uint8_t *codes_dev,
                             const float *scales_dev,
                             const uint16_t *tenants_dev, int64_t n,
                             void *stream);

/* Number of vectors in the index (for an id-map index: not deleted). */
tq_status tq_index_size(const tq_index *idx, int64_t *n_out);

/* Copies the index content back in the canonical layout: codes_dev
 * [n][d*bits/8], scales_dev [n], tenants_dev [n]; any may be NULL. */
tq_status tq_index_export(const tq_index *idx, uint8_t *codes_dev,
                          float *scales_dev, uint16_t *tenants_dev,
                          void *stream);

/* The index's d, bits, n_tenants, slot count n -- vectors ever added,
 * deleted ones included -- and whether it is an id-map index (1) or a
 * positional one (0); any output may be NULL. */
tq_status tq_index_info(const tq_index *idx, int32_t *d, int32_t *bits,
                        int32_t *n_tenants, int64_t *n, int32_t *idmap);

/* ------------------------------------------------------ TQ+ calibration ---
 * TQ+ (section II-B): a per-coordinate affine calibration for embeddings
 * whose rotated coordinates do not follow the sphere-coordinate law the
 * codebook was built for.  With y = R x / ||x|| (float64 from float32 R and
 * x), mu_j is the mean of y_j over a first batch of m rows and kappa_j =
 * sigma_j sqrt(d), sigma_j the population standard deviation (both stored
 * float32), so that z_j = (y_j - mu_j) / kappa_j has mean 0 and variance
 * 1/d over the batch.  Coordinates are then coded against per-coordinate
 * thresholds and reconstructed affinely; for a vector with n_x = ||x||:
 *   a_ij   = fl64(mu_j + fl64(kappa_j t_i))                (float64)
 *   code_j = number of i with fl64(a_ij * n_x) <= (R x)_j
 *   yhat_j = fl64(mu_j + fl64(kappa_j c[code_j]))
 *   scale  = n_x / sqrt(sum_j fl64(yhat_j^2))   (sequential over j; 0 if n_x = 0)
 * and a search scores scale * sum_j q'_j (mu_j + kappa_j c[code_j]).  The
 * identity calibration (mu = 0, kappa = 1) gives plain TurboQuant.
 *
 * calibrate(): fits mu and kappa to X_dev [m][d] float32 (m >= 1; sums in
 * float64 on the device) and installs them.  Only on an index with no
 * vectors (TQ_EINVAL otherwise, or for a row of zero or non-finite norm,
 * reported after synchronising `stream`).  Vectors added afterwards -- by
 * tq_index_add / tq_index_add_ids -- are coded as above; codes given to
 * tq_index_add_codes are taken to be calibrated codes.
 * set_calibration(): installs host mu [d], kappa [d] (finite, kappa >= 0)
 * on an index with no vectors.
 * calibration(): copies the installed values to mu_host, kappa_host (either
 * may be NULL) and sets *calibrated to 1, or sets it to 0 and copies nothing.
 * A calibrated index is searched by the scans only: TQ_PATH_MFMA is
 * TQ_EUNSUPPORTED on it. */
tq_status tq_index_calibrate(tq_index *idx, const float *X_dev, int64_t m, void *stream);
tq_status tq_index_set_calibration(tq_index *idx, const float *mu_host, const float *kappa_host);
tq_status tq_index_calibration(const tq_index *idx, float *mu_host, float *kappa_host,
                               int32_t *calibrated);

/* Persistence (section III-A: both index types persist to disk).
 * save() writes the index to `path` (created or truncated): a 48-byte header
 * (magic "TQINDEX1", format version 1, flags, d, bits, rotation seed, n,
 * n_tenants), the canonical codes [n][d*bits/8], the scales [n] float32 and
 * the tenant ids [n] uint16, then the optional sections the flags announce
 * (bit 0: an id-map index's ids and live masks, see below; bit 1: TQ+
 * calibration, mu [d] then kappa [d] float32), all little-endian, then a
 * 64-bit FNV-1a hash of every preceding byte.  The content is read back from the device with
 * blocking copies, and host memory of the file's size is used.  A file that
 * cannot be created or written is TQ_EINVAL. */
tq_status tq_index_save(const tq_index *idx, const char *path);

/* load() reads a file written by save() into a new index on the current
 * device, built on `cb` and `rot`; they must match the file's d, bits and
 * rotation seed (TQ_EINVAL otherwise).  The whole file is read and checked --
 * magic, header ranges, hash, no trailing bytes -- before any device work,
 * so a damaged or truncated file is TQ_EINVAL (TQ_EUNSUPPORTED for another
 * format version) and no index is made.  The caller frees *out with
 * tq_index_free.  Searches on the loaded index return what searches on the
 * saved one did. */
tq_status tq_index_load(const char *path, const tq_codebook *cb,
                        const tq_rotation *rot, tq_index **out);

void tq_index_free(tq_index *idx);

/* ---------------------------------------------------------- id-map index --
 * IdMapIndex (section III-A): the flat index of tq_index_create whose vectors
 * carry caller-chosen uint64 ids, with O(1) deletion and id-based access
 * control.  Vectors still occupy positions ("slots") in the store in the
 * order they are added; a deleted vector's slot stays, marked dead in its
 * block's live-slot mask, and the block's tenant summary is rebuilt over
 * its live slots, so deletions are folded into the block-skip test of the
 * scan (section III-B).  Searches return the external ids (uint64 bit
 * patterns in the int64 output; 2^64-1 is reserved, so -1 still marks
 * padding).  tq_index_add / tq_index_add_codes are TQ_EINVAL on it.  The
 * search, export, save and load calls work on both index types; an id-map
 * index with deleted vectors, or a search with a slot allowlist, always runs
 * the single-query scan (TQ_PATH_MFMA is TQ_EUNSUPPORTED then). */
tq_status tq_idmap_create(const tq_codebook *cb, const tq_rotation *rot,
                          int32_t n_tenants, tq_index **out);

/* As tq_index_add / tq_index_add_codes, with external ids ids_host [n]
 * (host memory).  Every id must be new to the index, distinct within the
 * call and not 2^64-1; otherwise TQ_EINVAL and nothing is added.
 * Synchronises `stream`. */
tq_status tq_index_add_ids(tq_index *idx, const float *X_dev,
                           const uint64_t *ids_host,
                           const uint16_t *tenants_dev, int64_t n,
                           void *stream);
tq_status tq_index_add_codes_ids(tq_index *idx, const uint8_t *codes_dev,
                                 const float *scales_dev,
                                 const uint64_t *ids_host,
                                 const uint16_t *tenants_dev, int64_t n,
                                 void *stream);

/* Deletes the vectors with ids ids_host [n] (host memory; ids not in the
 * index are ignored), each in O(1): the id leaves the host map, its slot's
 * live bit is cleared and its block's tenant summary is rebuilt.  A deleted
 * id may be added again (it gets a new slot).  *removed_out (may be NULL)
 * receives the number deleted.  Runs on the null stream and returns after
 * the device update; it must not overlap searches of the index. */
tq_status tq_index_remove_ids(tq_index *idx, const uint64_t *ids_host,
                              int64_t n, int64_t *removed_out);

/* The slot of each id in ids_host [n], or -1 when the index does not hold
 * it, into slots_host [n] (host memory).  On a positional index an id is its
 * slot (-1 past the end). */
tq_status tq_index_slots(const tq_index *idx, const uint64_t *ids_host,
                         int64_t n, int64_t *slots_host);

/* Slot-level allowlists (section III-B: access control by id).  Builds, for
 * nq queries, the bitmaps bitmap_dev [nq][ceil(n/64)] uint64 (n = the index's
 * slot count; slot v is bit v & 63 of word v >> 6) from the id lists
 * ids_host[offsets_host[q] .. offsets_host[q+1]) (host memory, offsets
 * [nq+1] starting at 0).  Ids the index does not hold are ignored.  Pass the
 * result to tq_search_ex with TQ_FLAG_SLOT_ALLOW; it is valid for the
 * index's current slot count.  Synchronises `stream`. */
tq_status tq_slot_allowlist(const tq_index *idx, const uint64_t *ids_host,
                            const int64_t *offsets_host, int64_t nq,
                            uint64_t *bitmap_dev, void *stream);

/* ------------------------------------------------------------ search ------
 * search(Q, k, allowlist) -> ids + scores -- section II-B step 5 and section
 * III-B.  For each query row q of Q_dev [nq][d] float32 (not normalised):
 *   score_i = scale_i * sum_j c[code_ij] * (R q)_j
 * over the vectors whose tenant bit is set in the query's allowlist row
 * allow_dev[q*W .. q*W+W) (uint64 words; tenant t is bit (t & 63) of word
 * t >> 6; allow_dev == NULL allows every vector).  64-vector blocks whose
 * tenant summary does not meet the allowlist are skipped before any of
 * their code bytes are read; disallowed vectors inside scanned blocks are
 * dropped at top-k insertion.
 * Output per query: the min(k, #allowed) best vectors ordered by (score
 * descending, id ascending) in ids_dev [nq][k] int64 and scores_dev [nq][k]
 * float32; unused slots hold id -1 and score -inf.
 * The search needs a device workspace; tq_search allocates it on `stream`
 * (stream-ordered allocation) and releases it before returning. */
tq_status tq_search(const tq_index *idx, const float *Q_dev, int64_t nq,
                    int32_t k, const uint64_t *allow_dev, int64_t *ids_dev,
                    float *scores_dev, void *stream);

/* Large k: for k <= 256 each wave of the scan keeps its best entries in
 * registers; for 256 < k <= 4096 the scan writes every vector's score (-inf
 * for filtered ones) to the workspace and a radix selection per query picks
 * the k best -- same scores, same order and tie rule. */

/* Over-fetch post-filter baseline (section V-C): the unfiltered top
 * k * overfetch of each query (k * overfetch <= 4096, else TQ_EUNSUPPORTED),
 * then, in that order, the first k vectors whose tenant the query's
 * allowlist row allow_dev[q*W .. q*W+W) admits; fewer than k leave padding
 * (-1, -inf).  This is the comparison method of the paper's filtered-search
 * study, not a filtered search: allowed vectors outside the over-fetched
 * list are missed.  Allocates its workspace on `stream` (stream-ordered). */
tq_status tq_search_postfilter(const tq_index *idx, const float *Q_dev,
                               int64_t nq, int32_t k, int32_t overfetch,
                               const uint64_t *allow_dev, int64_t *ids_dev,
                               float *scores_dev, void *stream);

/* Scan path selection for tq_search_ex (section II-B step 5; the batched
 * path is this library's, not the paper's).
 *  TQ_PATH_AUTO  the single-query scan.
 *  TQ_PATH_LUT   one pass over the code store per query, with the query's
 *                lookup table in LDS.
 *  TQ_PATH_MFMA  one pass per tile of 32 queries: approximate float16 scores
 *                on the matrix cores select 256 candidates per query (512
 *                for k > 64), which are rescored exactly (the same scores as
 *                TQ_PATH_LUT).  A
 *                per-query certificate -- a rigorous bound on the
 *                approximation error -- proves that the exact top k lies
 *                among the candidates; queries without one are re-run on the
 *                LUT path (see tq_last_search_fallbacks).  Needs 4-bit codes,
 *                d % 256 == 0, d <= 1792, k <= 256 and n_tenants <= 4096,
 *                else TQ_EUNSUPPORTED.  Synchronises `stream` once per call, to
 *                read the certificates on the host. */
typedef enum {
    TQ_PATH_AUTO = 0,
    TQ_PATH_LUT = 1,
    TQ_PATH_MFMA = 2
} tq_path;

/* Flag ORed into `path`: Q_dev already holds rotated queries R q (for
 * instance from tq_rotate_queries), so the rotation step is skipped. */
#define TQ_FLAG_PREROTATED 0x100

/* Flag ORed into `path`: allow_dev holds slot-level allowlists [nq][ceil(n/64)]
 * (see tq_slot_allowlist) instead of tenant allowlists: a vector may be
 * returned when its slot's bit is set.  Blocks with no allowed live slot are
 * skipped before their codes are read. */
#define TQ_FLAG_SLOT_ALLOW 0x200

/* Workspace size in bytes needed by tq_search_ex for (nq, k, path). */
tq_status tq_search_workspace_size(const tq_index *idx, int64_t nq, int32_t k,
                                   int32_t path, size_t *bytes_out);

/* tq_search with an explicit path and a caller-provided device workspace of
 * at least tq_search_workspace_size() bytes (256-byte aligned).  Allocates no
 * device memory.  Calls sharing one workspace must not overlap in time. */
tq_status tq_search_ex(const tq_index *idx, const float *Q_dev, int64_t nq,
                       int32_t k, const uint64_t *allow_dev, int32_t path,
                       void *workspace_dev, size_t workspace_bytes,
                       int64_t *ids_dev, float *scores_dev, void *stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): tq_search
 * with the same arguments, meaning, layout and results (the single-query
 * scan), whose workspace is a device array of TQ_NOALLOC_SCRATCH_BYTES held
 * by the library (one per GPU, kept until the process ends) instead of a
 * per-call allocation.  It calls no device allocation or free.
 * Queries are taken in as many consecutive launches as the array needs; a
 * search whose single query needs more than the array (k > 256 over a very
 * large index) returns TQ_EUNSUPPORTED.  The index's rotation must already
 * be on the current device -- it is uploaded by tq_index_reserve, the first
 * tq_index_add, tq_index_calibrate or allocating search on the index -- else
 * TQ_EINVAL.
 * Every call on one GPU shares that GPU's array: calls that overlap in time
 * on one GPU (two streams or threads) race and must be serialised by the
 * caller; consecutive calls on one stream are safe. */
#define TQ_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)
tq_status tq_search_noalloc(const tq_index *idx, const float *Q_dev, int64_t nq,
                            int32_t k, const uint64_t *allow_dev, int64_t *ids_dev,
                            float *scores_dev, void *stream);

/* Number of queries of the calling thread's last tq_search_ex call that the
 * TQ_PATH_MFMA path re-ran on the LUT path because their certificate failed
 * (0 after any other path). */
int32_t tq_last_search_fallbacks(void);

#ifdef __cplusplus
}
#endif

#endif /* TQ_H */
