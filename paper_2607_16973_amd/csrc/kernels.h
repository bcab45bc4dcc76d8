// Launch interface of the gfx950 kernels (host-callable, plain pointers).
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace tq {

// Fixed-size description of a codebook, passed to kernels by value.
struct CodebookDev {
    int bits;
    int levels;
    double bounds[255];   // levels-1 used
    float cents32[256];   // levels used
    double cent_sq[256];  // fl64(c * c), levels used
};

// ------------------------------------------------------------------ encode
// Rows per encode chunk and the workspace it needs.
constexpr int kEncodeChunkRows = 32768;
size_t encode_workspace_bytes(int d);

// Output layout selector for the encode pipeline.
struct EncodeOut {
    uint8_t *canonical = nullptr;   // [n][d*bits/8] canonical rows, or null
    float *scales = nullptr;        // [n] scales (canonical order), or null
    uint8_t *blocked = nullptr;     // index blocked code store, or null
    float *blocked_scales = nullptr;// index scale store, or null
    int64_t base = 0;               // index position of row 0 (blocked only)
};

// Encodes X [n][d] (float32, row-major) with R [d][d] on `stream`.
// `ws` must hold encode_workspace_bytes(d); `status_dev` is an int32 that the
// kernels set non-zero on a non-finite input.
// TQ+ calibration tables on the device (null: plain TurboQuant):
// athr [(levels-1)][d] per-coordinate thresholds mu_j + kappa_j t_i and ysq
// [d][levels] squares of the reconstructions mu_j + kappa_j c_c (float64).
struct CalibDev {
    const double *athr = nullptr;
    const double *ysq = nullptr;
};

hipError_t encode_rows(const float *X, int64_t n, int d, const float *R,
                       const CodebookDev &cb, const EncodeOut &out, void *ws,
                       int *status_dev, hipStream_t stream,
                       const CalibDev &calib = CalibDev());

// Y = X R^T in float32 (query rotation), X [m][d], Y [m][d].  With fill,
// the nfill ints at fill are also set to fill_value on the same stream (by
// the rotation's own launch when m <= 64), so that a search's first kernel
// can initialise its bounds without a launch of its own.
hipError_t rotate_rows_f32(const float *X, int64_t m, int d, const float *R,
                           float *Y, hipStream_t stream, int *fill = nullptr,
                           int64_t nfill = 0, int fill_value = 0);

// ------------------------------------------------------------- TQ+ (calib.hip)
// Fits mu [d] and kappa [d] (float32, device) to the m >= 1 rows of X:
// moments of the rotated, normalised rows.  `ws` holds
// calib_workspace_bytes(d); *status_dev gets bit 0 set when a row has a zero
// or non-finite norm.
size_t calib_workspace_bytes(int d);
hipError_t calib_fit(const float *X, int64_t m, int d, const float *R, void *ws, int *status_dev,
                     float *mu, float *kappa, hipStream_t stream);
// Qout = kappa * Qin per row (Qout may be Qin) and qconst [nq] = sum_j mu_j
// Qin_j: the query form the scans take for a calibrated index.
hipError_t calib_queries(const float *Qin, int64_t nq, int d, const float *mu, const float *kappa,
                         float *Qout, float *qconst, hipStream_t stream);

// --------------------------------------------------------------- layout
// Blocked code store: vector v lives in block v/64, lane v%64; chunk c (16 B)
// of a vector sits at byte ((v/64) * chunks + c) * 1024 + (v%64) * 16.
// For b in {1, 2, 4} every 32-bit word of a chunk holds the canonical word
// rotated left by 2 bits (field t of 4 bits at bits [4t+2, 4t+6) mod 32), so
// the scan gets each 4-bit field times 4 in a byte with one mask per half.
__host__ __device__ inline bool blocked_rotated(int bits) { return bits == 1 || bits == 2 || bits == 4; }
__host__ __device__ inline uint32_t rotl2(uint32_t w) { return (w << 2) | (w >> 30); }
__host__ __device__ inline uint32_t rotr2(uint32_t w) { return (w >> 2) | (w << 30); }
inline int chunks_per_vector(int d, int bits) {
    // 3-bit codes are stored 10 per 32-bit word (2 pad bits per word), in a
    // whole number of 4-chunk groups (zero codes past d) so the scan can keep
    // at least 4 chunk loads in flight
    if (bits == 3) return ((((d + 9) / 10) + 3) / 4 + 3) / 4 * 4;
    return d * bits / 128;
}

hipError_t canonical_to_blocked(const uint8_t *canon, const float *scales,
                                int64_t n, int d, int bits, uint8_t *blocked,
                                float *blocked_scales, int64_t base,
                                hipStream_t stream);
hipError_t blocked_to_canonical(const uint8_t *blocked, const float *blocked_scales,
                                int64_t n, int d, int bits, uint8_t *canon,
                                float *scales, hipStream_t stream);
// Copies tenant ids into the store and ORs them into the block summaries
// (W words per block); sets *status_dev non-zero if an id is >= n_tenants.
hipError_t add_tenants(const uint16_t *tenants, int64_t n, int64_t base,
                       int n_tenants, int W, uint16_t *tenant_store,
                       uint64_t *summaries, int *status_dev, hipStream_t stream);

// IdMapIndex support (layout.hip).  set_live marks slots [base, base+n)
// live; retire_slots clears, for each listed block, the slots of its `clear`
// mask and rebuilds the block's tenant summary over its live slots (W <=
// 1024); map_ids replaces slot ids >= 0 by ext[slot].
hipError_t set_live(uint64_t *live, int64_t base, int64_t n, hipStream_t stream);
hipError_t retire_slots(const int64_t *blocks, const uint64_t *clear, int64_t nb, uint64_t *live,
                        const uint16_t *tenants, int W, uint64_t *summaries, hipStream_t stream);
hipError_t map_ids(int64_t *ids, int64_t count, const uint64_t *ext, hipStream_t stream);

// Over-fetch post-filter: from lists of kk (slot id, score) in rank order,
// the first k whose tenant the query's allowlist row admits.
hipError_t postfilter(const int64_t *ids_in, const float *sc_in, int64_t nq, int kk,
                      const uint16_t *tenants, const uint64_t *allow, int W, int k,
                      int64_t *ids_out, float *sc_out, hipStream_t stream);

// ----------------------------------------------------------------- search
struct ScanShape {
    int d, bits, chunks;     // code geometry
    int64_t n;               // vectors in the index
    int64_t nblk;            // 64-vector blocks
    int W;                   // allowlist words per query
};

// Largest k of the per-wave top-k scans; larger k (up to kMaxK) scores every
// vector and selects per query.
constexpr int kMaxTopK = 256;
constexpr int kMaxK = 4096;

size_t lut_search_workspace_bytes(const ScanShape &s, int64_t nq, int k, int grid);
// Which slots a search may return: tenant allowlists [nq][W] (null: every
// tenant), per-block live-slot masks [nblk] (null: no slot deleted) and
// per-query slot allowlists [nq][nblk] (null: none).  Any non-null member
// sends the search through the filtered scans.
struct SearchFilter {
    const uint64_t *allow = nullptr;
    const uint64_t *live = nullptr;
    const uint64_t *slot_allow = nullptr;
    bool any() const { return allow || live || slot_allow; }
};

// qconst: [nq] constant terms of TQ+ calibrated scores (Qrot then holds
// kappa * q'), or null.  bounds_ready: the queries' global bounds (at
// lut_search_bounds) already hold kBoundInit.
hipError_t lut_search(const ScanShape &s, const uint8_t *blocked, const float *scales,
                      const uint16_t *tenants, const uint64_t *summaries,
                      const float *cents32, const float *Qrot, int64_t nq, int k,
                      const SearchFilter &filter, int grid, void *ws, size_t ws_bytes,
                      int64_t *ids, float *scores, hipStream_t stream,
                      const float *qconst = nullptr, bool bounds_ready = false);
// The order key of -inf: the value the global bounds of a top-k search
// start from.
constexpr int kBoundInit = (int)0x807FFFFFu;
// Where lut_search keeps the queries' global bounds (nq ints) when it runs
// the top-k path in one query chunk, else null.  A search sets them to
// kBoundInit ahead of the scan (in the query rotation's launch) and passes
// bounds_ready = true, so that the scan's launch follows the rotation
// without a launch of its own in between.
int *lut_search_bounds(const ScanShape &s, int64_t nq, int k, int grid, void *ws);

// Batched search of a tile of queries on the matrix cores with exact
// rescoring (b = 4, chunks % 8 == 0, d <= 1792, k <= 256, at most 4096
// tenants).
// cmax16 = max |float16(c_l)|, dmax = max |float16(c_l) - c_l| over the
// float32 centroids cents32.
// Queries whose top k the certificate does not prove are re-run on the
// single-query scan; their count goes to *n_fallback.  Synchronises
// `stream` once to read the certificates.  `smax` is a device float: the
// largest scale in the store.
bool mfma_search_supported(const ScanShape &s, int k);
size_t mfma_search_workspace_bytes(const ScanShape &s, int64_t nq, int k, int grid);
hipError_t mfma_search(const ScanShape &s, const uint8_t *blocked, const float *scales,
                       const float *smax, const uint16_t *tenants, const uint64_t *summaries,
                       const float *cents32, float cmax16, float dmax, const float *Qrot,
                       int64_t nq, int k,
                       const uint64_t *allow, int grid, void *ws, int64_t *ids, float *scores,
                       int *n_fallback, hipStream_t stream);
// *smax = max(*smax, max of scales[0..n)); scales are >= 0.
hipError_t update_scale_max(const float *scales, int64_t n, float *smax, hipStream_t stream);

int device_cu_count();

}  // namespace tq
