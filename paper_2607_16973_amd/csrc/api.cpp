// C ABI of libtq: argument validation, handles, device storage, dispatch.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <new>
#include <string>
#include <unordered_map>
#include <vector>

#include "kernels.h"
#include "tq_internal.h"

namespace tq {

namespace {
thread_local std::string g_err;
// queries of the calling thread's last search that the matrix-core path
// handed to the single-query scan
thread_local int g_last_fallbacks = 0;

bool valid_bits(int b) { return b == 1 || b == 2 || b == 3 || b == 4 || b == 8; }

tq_status check_d(int32_t d) {
    if (d < 64 || d > 2048 || d % 64 != 0)
        return fail(TQ_EINVAL, "d must be a multiple of 64 in [64, 2048], got " + std::to_string(d));
    return TQ_OK;
}

tq_status check_geometry(int32_t d, int32_t bits) {
    tq_status st = check_d(d);
    if (st != TQ_OK) return st;
    if (!valid_bits(bits))
        return fail(TQ_EUNSUPPORTED, "bits must be one of 1, 2, 3, 4, 8; got " + std::to_string(bits));
    if ((bits == 1 || bits == 3) && d % 128 != 0)
        return fail(TQ_EINVAL, "bits = 1 or 3 needs d % 128 == 0");
    return TQ_OK;
}

tq_status device_ready() {
    int n = 0;
    hipError_t e = hipGetDeviceCount(&n);
    if (e != hipSuccess || n <= 0) {
        (void)hipGetLastError();
        return fail(TQ_EDEVICE, "no usable GPU (hipGetDeviceCount: " +
                                    std::string(hipGetErrorString(e)) + ")");
    }
    return TQ_OK;
}

tq_status hip_fail(hipError_t e, const char *what) {
    (void)hipGetLastError();
    if (e == hipErrorOutOfMemory)
        return fail(TQ_ENOMEM, std::string(what) + ": out of device memory");
    return fail(TQ_EDEVICE, std::string(what) + ": " + hipGetErrorString(e));
}

void fill_codebook_dev(const CodebookTables &t, CodebookDev *cd) {
    std::memset(cd, 0, sizeof(*cd));
    cd->bits = t.bits;
    cd->levels = 1 << t.bits;
    for (int i = 0; i < cd->levels - 1; ++i) cd->bounds[i] = t.bounds[i];
    for (int i = 0; i < cd->levels; ++i) {
        cd->cents32[i] = (float)t.cents[i];
        const double c = t.cents[i];
        const double sq = c * c;
        cd->cent_sq[i] = sq;
    }
}

// Device copy of the rotation matrix on the current device.
tq_status rotation_dev(const tq_rotation *rot, const float **out) {
    std::lock_guard<std::mutex> lk(rot->mu);
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (rot->R_dev && rot->R_dev_device == dev) {
        *out = rot->R_dev;
        return TQ_OK;
    }
    if (rot->R_dev) {
        (void)hipFree(rot->R_dev);
        rot->R_dev = nullptr;
    }
    const size_t bytes = sizeof(float) * rot->R.size();
    e = hipMalloc(&rot->R_dev, bytes);
    if (e != hipSuccess) return hip_fail(e, "hipMalloc(rotation)");
    e = hipMemcpy(rot->R_dev, rot->R.data(), bytes, hipMemcpyHostToDevice);
    if (e != hipSuccess) return hip_fail(e, "hipMemcpy(rotation)");
    rot->R_dev_device = dev;
    *out = rot->R_dev;
    return TQ_OK;
}

// Stream-ordered scratch allocation released on destruction.
// Device scratch released on destruction (synchronous allocation).
struct DevBuf {
    void *p = nullptr;
    hipError_t alloc(size_t bytes) { return hipMalloc(&p, bytes ? bytes : 1); }
    ~DevBuf() {
        if (p) (void)hipFree(p);
    }
};

struct AsyncBuf {
    void *p = nullptr;
    hipStream_t s = nullptr;
    hipError_t alloc(size_t bytes, hipStream_t stream) {
        s = stream;
        return hipMallocAsync(&p, bytes, stream);
    }
    ~AsyncBuf() {
        if (p) (void)hipFreeAsync(p, s);
    }
};

}  // namespace

void set_error(const std::string &msg) { g_err = msg; }

tq_status fail(tq_status st, const std::string &msg) {
    g_err = msg;
    return st;
}

}  // namespace tq

using namespace tq;

struct tq_index {
    CodebookTables cb;
    CodebookDev cbdev;
    tq_rotation rot;
    int d = 0, bits = 0, T = 0, W = 0, chunks = 0;
    int64_t n = 0, cap = 0;
    uint8_t *codes = nullptr;      // blocked store, cap/64 blocks
    float *scales = nullptr;       // cap
    uint16_t *tenants = nullptr;   // cap
    uint64_t *summ = nullptr;      // cap/64 * W
    float *cents_dev = nullptr;    // levels
    int *status = nullptr;         // device status word
    int device = -1;
    // IdMapIndex (section III-A): the external id of every slot and the
    // live-slot mask of every block on the device, the map from external id
    // to slot on the host.  Deleted slots stay in the store, dead.
    bool idmap = false;
    uint64_t *ext = nullptr;       // cap
    uint64_t *live = nullptr;      // cap/64
    std::unordered_map<uint64_t, int64_t> slot_of;
    int64_t n_deleted = 0;
    // TQ+ calibration (section II-B): mu and kappa per coordinate (host and
    // device float32) and the encoder's float64 tables derived from them.
    bool calibrated = false;
    std::vector<float> mu_h, kappa_h;
    float *mu = nullptr, *kappa = nullptr;   // [d] each
    double *athr = nullptr;                  // [levels-1][d]: mu_j + kappa_j t_i
    double *ysq = nullptr;                   // [d][levels]: (mu_j + kappa_j c_c)^2
};

namespace tq {

// Whether the index's rotation is already on the current device, so that a
// search rotates its queries without allocating.
bool index_rotation_resident(const tq_index *x) {
    std::lock_guard<std::mutex> lk(x->rot.mu);
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) {
        (void)hipGetLastError();
        return false;
    }
    return x->rot.R_dev != nullptr && x->rot.R_dev_device == dev;
}

}  // namespace tq

namespace {

size_t block_bytes(const tq_index *x) { return (size_t)x->chunks * 1024; }

// The device status buffer (256 bytes) holds the status word at byte 0 and
// the largest scale in the store, a float, at byte 64.
float *scale_max_dev(const tq_index *x) { return reinterpret_cast<float *>(x->status) + 16; }

void index_release(tq_index *x) {
    if (x->codes) (void)hipFree(x->codes);
    if (x->scales) (void)hipFree(x->scales);
    if (x->tenants) (void)hipFree(x->tenants);
    if (x->summ) (void)hipFree(x->summ);
    if (x->cents_dev) (void)hipFree(x->cents_dev);
    if (x->status) (void)hipFree(x->status);
    if (x->ext) (void)hipFree(x->ext);
    if (x->live) (void)hipFree(x->live);
    if (x->mu) (void)hipFree(x->mu);
    if (x->kappa) (void)hipFree(x->kappa);
    if (x->athr) (void)hipFree(x->athr);
    if (x->ysq) (void)hipFree(x->ysq);
    x->mu = x->kappa = nullptr;
    x->athr = x->ysq = nullptr;
    x->calibrated = false;
    x->ext = nullptr;
    x->live = nullptr;
    x->codes = nullptr;
    x->scales = nullptr;
    x->tenants = nullptr;
    x->summ = nullptr;
    x->cents_dev = nullptr;
    x->status = nullptr;
}

tq_status index_device_init(tq_index *x) {
    if (x->cents_dev) return TQ_OK;
    tq_status st = device_ready();
    if (st != TQ_OK) return st;
    hipError_t e = hipGetDevice(&x->device);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    e = hipMalloc(&x->cents_dev, sizeof(float) * 256);
    if (e != hipSuccess) return hip_fail(e, "hipMalloc(centroids)");
    e = hipMemcpy(x->cents_dev, x->cbdev.cents32, sizeof(float) * 256, hipMemcpyHostToDevice);
    if (e != hipSuccess) return hip_fail(e, "hipMemcpy(centroids)");
    e = hipMalloc(&x->status, 256);
    if (e != hipSuccess) return hip_fail(e, "hipMalloc(status)");
    e = hipMemset(x->status, 0, 256);
    if (e != hipSuccess) return hip_fail(e, "hipMemset(status)");
    return TQ_OK;
}

tq_status index_grow(tq_index *x, int64_t need, hipStream_t stream) {
    tq_status st = index_device_init(x);
    if (st != TQ_OK) return st;
    if (need <= x->cap) return TQ_OK;
    int64_t cap = std::max<int64_t>(need, x->cap + x->cap / 2);
    cap = (cap + 63) / 64 * 64;
    const int64_t nb = cap / 64;
    uint8_t *codes = nullptr;
    float *scales = nullptr;
    uint16_t *ten = nullptr;
    uint64_t *summ = nullptr, *ext = nullptr, *live = nullptr;
    auto free_new = [&]() {
        if (codes) (void)hipFree(codes);
        if (scales) (void)hipFree(scales);
        if (ten) (void)hipFree(ten);
        if (summ) (void)hipFree(summ);
        if (ext) (void)hipFree(ext);
        if (live) (void)hipFree(live);
    };
    hipError_t e;
    if ((e = hipMalloc(&codes, nb * block_bytes(x))) != hipSuccess ||
        (e = hipMalloc(&scales, cap * sizeof(float))) != hipSuccess ||
        (e = hipMalloc(&ten, cap * sizeof(uint16_t))) != hipSuccess ||
        (e = hipMalloc(&summ, nb * x->W * sizeof(uint64_t))) != hipSuccess ||
        (x->idmap && (e = hipMalloc(&ext, cap * sizeof(uint64_t))) != hipSuccess) ||
        (x->idmap && (e = hipMalloc(&live, nb * sizeof(uint64_t))) != hipSuccess)) {
        free_new();
        return hip_fail(e, "hipMalloc(index storage)");
    }
    e = hipMemsetAsync(codes, 0, nb * block_bytes(x), stream);
    if (e == hipSuccess) e = hipMemsetAsync(scales, 0, cap * sizeof(float), stream);
    if (e == hipSuccess) e = hipMemsetAsync(ten, 0, cap * sizeof(uint16_t), stream);
    if (e == hipSuccess) e = hipMemsetAsync(summ, 0, nb * x->W * sizeof(uint64_t), stream);
    if (e == hipSuccess && live) e = hipMemsetAsync(live, 0, nb * sizeof(uint64_t), stream);
    if (e == hipSuccess && x->cap > 0) {
        const int64_t ob = x->cap / 64;
        e = hipMemcpyAsync(codes, x->codes, ob * block_bytes(x), hipMemcpyDeviceToDevice, stream);
        if (e == hipSuccess)
            e = hipMemcpyAsync(scales, x->scales, x->cap * sizeof(float), hipMemcpyDeviceToDevice, stream);
        if (e == hipSuccess)
            e = hipMemcpyAsync(ten, x->tenants, x->cap * sizeof(uint16_t), hipMemcpyDeviceToDevice, stream);
        if (e == hipSuccess)
            e = hipMemcpyAsync(summ, x->summ, ob * x->W * sizeof(uint64_t), hipMemcpyDeviceToDevice, stream);
        if (e == hipSuccess && ext)
            e = hipMemcpyAsync(ext, x->ext, x->cap * sizeof(uint64_t), hipMemcpyDeviceToDevice, stream);
        if (e == hipSuccess && live)
            e = hipMemcpyAsync(live, x->live, ob * sizeof(uint64_t), hipMemcpyDeviceToDevice, stream);
    }
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    if (e != hipSuccess) {
        free_new();
        return hip_fail(e, "index growth");
    }
    if (x->codes) (void)hipFree(x->codes);
    if (x->scales) (void)hipFree(x->scales);
    if (x->tenants) (void)hipFree(x->tenants);
    if (x->summ) (void)hipFree(x->summ);
    if (x->ext) (void)hipFree(x->ext);
    if (x->live) (void)hipFree(x->live);
    x->codes = codes;
    x->scales = scales;
    x->tenants = ten;
    x->summ = summ;
    x->ext = ext;
    x->live = live;
    x->cap = cap;
    return TQ_OK;
}

tq_status read_status(int *status_dev, hipStream_t stream, int *out) {
    int h = 0;
    hipError_t e = hipMemcpyAsync(&h, status_dev, sizeof(int), hipMemcpyDeviceToHost, stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    if (e != hipSuccess) return hip_fail(e, "status read");
    *out = h;
    return TQ_OK;
}

}  // namespace

extern "C" {

const char *tq_last_error(void) { return g_err.c_str(); }

const char *tq_version(void) { return "tq 0.1.0 gfx950"; }

int32_t tq_last_search_fallbacks(void) { return g_last_fallbacks; }

tq_status tq_build_codebook(int32_t d, int32_t bits, tq_codebook **out) {
    if (!out) return fail(TQ_EINVAL, "out is NULL");
    *out = nullptr;
    tq_status st = check_geometry(d, bits);
    if (st != TQ_OK) return st;
    tq_codebook *cb = new (std::nothrow) tq_codebook();
    if (!cb) return fail(TQ_ENOMEM, "host allocation failed");
    if (!solve_lloyd_max(d, bits, &cb->t)) {
        delete cb;
        return TQ_EINVAL;
    }
    *out = cb;
    return TQ_OK;
}

tq_status tq_codebook_tables(const tq_codebook *cb, double *bounds_host, double *cents_host) {
    if (!cb) return fail(TQ_EINVAL, "codebook is NULL");
    if (bounds_host) std::memcpy(bounds_host, cb->t.bounds.data(), cb->t.bounds.size() * sizeof(double));
    if (cents_host) std::memcpy(cents_host, cb->t.cents.data(), cb->t.cents.size() * sizeof(double));
    return TQ_OK;
}

tq_status tq_codebook_mse(const tq_codebook *cb, double *mse_out) {
    if (!cb || !mse_out) return fail(TQ_EINVAL, "NULL argument");
    *mse_out = cb->t.mse;
    return TQ_OK;
}

void tq_codebook_free(tq_codebook *cb) { delete cb; }

tq_status tq_rotation_create(int32_t d, uint64_t seed, tq_rotation **out) {
    if (!out) return fail(TQ_EINVAL, "out is NULL");
    *out = nullptr;
    tq_status st = check_d(d);
    if (st != TQ_OK) return st;
    tq_rotation *r = new (std::nothrow) tq_rotation();
    if (!r) return fail(TQ_ENOMEM, "host allocation failed");
    r->d = d;
    r->seed = seed;
    try {
        make_rotation(d, seed, &r->R);
    } catch (const std::bad_alloc &) {
        delete r;
        return fail(TQ_ENOMEM, "host allocation failed");
    }
    *out = r;
    return TQ_OK;
}

tq_status tq_rotation_matrix(const tq_rotation *rot, float *R_host) {
    if (!rot || !R_host) return fail(TQ_EINVAL, "NULL argument");
    std::memcpy(R_host, rot->R.data(), rot->R.size() * sizeof(float));
    return TQ_OK;
}

void tq_rotation_free(tq_rotation *rot) {
    if (!rot) return;
    if (rot->R_dev) (void)hipFree(rot->R_dev);
    delete rot;
}

tq_status tq_rotate_quantize(const tq_codebook *cb, const tq_rotation *rot, const float *X_dev,
                             int64_t n, uint8_t *codes_dev, float *scales_dev, void *stream) {
    if (!cb || !rot) return fail(TQ_EINVAL, "NULL codebook or rotation");
    if (n < 0) return fail(TQ_EINVAL, "n < 0");
    if (cb->t.d != rot->d) return fail(TQ_EINVAL, "codebook and rotation disagree on d");
    if (n == 0) return TQ_OK;
    if (!X_dev || !codes_dev || !scales_dev) return fail(TQ_EINVAL, "NULL device pointer");
    tq_status st = device_ready();
    if (st != TQ_OK) return st;
    const float *R = nullptr;
    st = rotation_dev(rot, &R);
    if (st != TQ_OK) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    CodebookDev cd;
    fill_codebook_dev(cb->t, &cd);
    const int d = rot->d;
    AsyncBuf ws;
    hipError_t e = ws.alloc(encode_workspace_bytes(d) + 256, s);
    if (e != hipSuccess) return hip_fail(e, "hipMallocAsync(encode workspace)");
    int *status = reinterpret_cast<int *>(static_cast<uint8_t *>(ws.p) + encode_workspace_bytes(d));
    e = hipMemsetAsync(status, 0, sizeof(int), s);
    if (e != hipSuccess) return hip_fail(e, "hipMemsetAsync");
    EncodeOut out;
    out.canonical = codes_dev;
    out.scales = scales_dev;
    e = encode_rows(X_dev, n, d, R, cd, out, ws.p, status, s);
    if (e != hipSuccess) return hip_fail(e, "encode");
    int h = 0;
    st = read_status(status, s, &h);
    if (st != TQ_OK) return st;
    if (h & 1) return fail(TQ_EINVAL, "non-finite value in X");
    return TQ_OK;
}

tq_status tq_rotate_queries(const tq_rotation *rot, const float *Q_dev, int64_t nq,
                            float *Qrot_dev, void *stream) {
    if (!rot) return fail(TQ_EINVAL, "NULL rotation");
    if (nq < 0) return fail(TQ_EINVAL, "nq < 0");
    if (nq == 0) return TQ_OK;
    if (!Q_dev || !Qrot_dev) return fail(TQ_EINVAL, "NULL device pointer");
    tq_status st = device_ready();
    if (st != TQ_OK) return st;
    const float *R = nullptr;
    st = rotation_dev(rot, &R);
    if (st != TQ_OK) return st;
    hipError_t e = rotate_rows_f32(Q_dev, nq, rot->d, R, Qrot_dev, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "query rotation");
    return TQ_OK;
}

tq_status tq_index_create(const tq_codebook *cb, const tq_rotation *rot, int32_t n_tenants,
                          tq_index **out) {
    if (!out) return fail(TQ_EINVAL, "out is NULL");
    *out = nullptr;
    if (!cb || !rot) return fail(TQ_EINVAL, "NULL codebook or rotation");
    if (cb->t.d != rot->d) return fail(TQ_EINVAL, "codebook and rotation disagree on d");
    if (n_tenants < 1 || n_tenants > 65535) return fail(TQ_EINVAL, "n_tenants must be in 1..65535");
    tq_index *x = new (std::nothrow) tq_index();
    if (!x) return fail(TQ_ENOMEM, "host allocation failed");
    x->cb = cb->t;
    fill_codebook_dev(x->cb, &x->cbdev);
    x->rot.d = rot->d;
    x->rot.seed = rot->seed;
    x->rot.R = rot->R;
    x->d = rot->d;
    x->bits = cb->t.bits;
    x->T = n_tenants;
    x->W = (n_tenants + 63) / 64;
    x->chunks = chunks_per_vector(x->d, x->bits);
    *out = x;
    return TQ_OK;
}

tq_status tq_index_reserve(tq_index *idx, int64_t capacity) {
    if (!idx) return fail(TQ_EINVAL, "NULL index");
    if (capacity < 0) return fail(TQ_EINVAL, "capacity < 0");
    tq_status st = index_grow(idx, capacity, nullptr);
    if (st != TQ_OK) return st;
    // the encoder's copy of the rotation on the current device (otherwise
    // uploaded by the first add)
    const float *R = nullptr;
    return rotation_dev(&idx->rot, &R);
}

static tq_status finish_add(tq_index *x, const uint16_t *tenants_dev, int64_t n, hipStream_t s) {
    hipError_t e = hipMemsetAsync(x->status, 0, sizeof(int), s);
    if (e != hipSuccess) return hip_fail(e, "hipMemsetAsync");
    e = add_tenants(tenants_dev, n, x->n, x->T, x->W, x->tenants, x->summ, x->status, s);
    if (e != hipSuccess) return hip_fail(e, "add_tenants");
    e = update_scale_max(x->scales + x->n, n, scale_max_dev(x), s);
    if (e != hipSuccess) return hip_fail(e, "scale maximum");
    int h = 0;
    tq_status st = read_status(x->status, s, &h);
    if (st != TQ_OK) return st;
    if (h & 2) return fail(TQ_EINVAL, "tenant id >= n_tenants");
    x->n += n;
    return TQ_OK;
}

static tq_status add_vectors(tq_index *idx, const float *X_dev, const uint16_t *tenants_dev,
                             int64_t n, void *stream) {
    if (!X_dev) return fail(TQ_EINVAL, "NULL device pointer");
    if (idx->n + n > (int64_t)INT32_MAX) return fail(TQ_EUNSUPPORTED, "index limited to 2^31-1 vectors");
    hipStream_t s = static_cast<hipStream_t>(stream);
    tq_status st = index_grow(idx, idx->n + n, s);
    if (st != TQ_OK) return st;
    const float *R = nullptr;
    st = rotation_dev(&idx->rot, &R);
    if (st != TQ_OK) return st;
    AsyncBuf ws;
    hipError_t e = ws.alloc(encode_workspace_bytes(idx->d), s);
    if (e != hipSuccess) return hip_fail(e, "hipMallocAsync(encode workspace)");
    e = hipMemsetAsync(idx->status, 0, sizeof(int), s);
    if (e != hipSuccess) return hip_fail(e, "hipMemsetAsync");
    EncodeOut out;
    out.blocked = idx->codes;
    out.blocked_scales = idx->scales;
    out.base = idx->n;
    CalibDev cal;
    if (idx->calibrated) {
        cal.athr = idx->athr;
        cal.ysq = idx->ysq;
    }
    e = encode_rows(X_dev, n, idx->d, R, idx->cbdev, out, ws.p, idx->status, s, cal);
    if (e != hipSuccess) return hip_fail(e, "encode");
    int h = 0;
    st = read_status(idx->status, s, &h);
    if (st != TQ_OK) return st;
    if (h & 1) return fail(TQ_EINVAL, "non-finite value in X");
    return finish_add(idx, tenants_dev, n, s);
}

static tq_status add_codes_impl(tq_index *idx, const uint8_t *codes_dev, const float *scales_dev,
                                const uint16_t *tenants_dev, int64_t n, void *stream) {
    if (!codes_dev || !scales_dev) return fail(TQ_EINVAL, "NULL device pointer");
    if (idx->n + n > (int64_t)INT32_MAX) return fail(TQ_EUNSUPPORTED, "index limited to 2^31-1 vectors");
    hipStream_t s = static_cast<hipStream_t>(stream);
    tq_status st = index_grow(idx, idx->n + n, s);
    if (st != TQ_OK) return st;
    hipError_t e = canonical_to_blocked(codes_dev, scales_dev, n, idx->d, idx->bits, idx->codes,
                                        idx->scales, idx->n, s);
    if (e != hipSuccess) return hip_fail(e, "canonical_to_blocked");
    return finish_add(idx, tenants_dev, n, s);
}

tq_status tq_index_add(tq_index *idx, const float *X_dev, const uint16_t *tenants_dev, int64_t n,
                       void *stream) {
    if (!idx) return fail(TQ_EINVAL, "NULL index");
    if (idx->idmap) return fail(TQ_EINVAL, "an id-map index takes vectors with ids (tq_index_add_ids)");
    if (n < 0) return fail(TQ_EINVAL, "n < 0");
    if (n == 0) return TQ_OK;
    return add_vectors(idx, X_dev, tenants_dev, n, stream);
}

tq_status tq_index_add_codes(tq_index *idx, const uint8_t *codes_dev, const float *scales_dev,
                             const uint16_t *tenants_dev, int64_t n, void *stream) {
    if (!idx) return fail(TQ_EINVAL, "NULL index");
    if (idx->idmap) return fail(TQ_EINVAL, "an id-map index takes vectors with ids (tq_index_add_codes_ids)");
    if (n < 0) return fail(TQ_EINVAL, "n < 0");
    if (n == 0) return TQ_OK;
    return add_codes_impl(idx, codes_dev, scales_dev, tenants_dev, n, stream);
}

tq_status tq_idmap_create(const tq_codebook *cb, const tq_rotation *rot, int32_t n_tenants,
                          tq_index **out) {
    tq_status st = tq_index_create(cb, rot, n_tenants, out);
    if (st == TQ_OK) (*out)->idmap = true;
    return st;
}

}  // extern "C"

// Installs a TQ+ calibration (host mu, kappa; checked finite, kappa >= 0):
// the device copies and the encoder's tables, thresholds a_ij =
// fl64(mu_j + fl64(kappa_j t_i)) and squared reconstructions
// fl64(fl64(mu_j + fl64(kappa_j c_c))^2), each operation rounded on its own.
static tq_status install_calibration(tq_index *x, const float *mu, const float *kappa) {
    const int d = x->d, L = 1 << x->bits;
    for (int j = 0; j < d; ++j)
        if (!std::isfinite(mu[j]) || !std::isfinite(kappa[j]) || kappa[j] < 0.f)
            return fail(TQ_EINVAL, "calibration values must be finite, kappa >= 0");
    tq_status st = index_device_init(x);
    if (st != TQ_OK) return st;
    std::vector<double> athr((size_t)(L - 1) * d), ysq((size_t)d * L);
    for (int i = 0; i < L - 1; ++i)
        for (int j = 0; j < d; ++j) {
            const double p = (double)kappa[j] * x->cb.bounds[i];
            const double a = (double)mu[j] + p;
            athr[(size_t)i * d + j] = a;
        }
    for (int j = 0; j < d; ++j)
        for (int c = 0; c < L; ++c) {
            const double p = (double)kappa[j] * x->cb.cents[c];
            const double y = (double)mu[j] + p;
            const double y2 = y * y;
            ysq[(size_t)j * L + c] = y2;
        }
    if (!x->mu) {
        hipError_t e = hipMalloc(&x->mu, sizeof(float) * d);
        if (e == hipSuccess) e = hipMalloc(&x->kappa, sizeof(float) * d);
        if (e == hipSuccess) e = hipMalloc(&x->athr, sizeof(double) * athr.size());
        if (e == hipSuccess) e = hipMalloc(&x->ysq, sizeof(double) * ysq.size());
        if (e != hipSuccess) return hip_fail(e, "hipMalloc(calibration)");
    }
    hipError_t e = hipMemcpy(x->mu, mu, sizeof(float) * d, hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemcpy(x->kappa, kappa, sizeof(float) * d, hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemcpy(x->athr, athr.data(), sizeof(double) * athr.size(), hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemcpy(x->ysq, ysq.data(), sizeof(double) * ysq.size(), hipMemcpyHostToDevice);
    if (e != hipSuccess) return hip_fail(e, "calibration upload");
    x->mu_h.assign(mu, mu + d);
    x->kappa_h.assign(kappa, kappa + d);
    x->calibrated = true;
    return TQ_OK;
}

extern "C" {

tq_status tq_index_calibrate(tq_index *idx, const float *X_dev, int64_t m, void *stream) {
    if (!idx) return fail(TQ_EINVAL, "NULL index");
    if (idx->n != 0) return fail(TQ_EINVAL, "calibration must precede the first vector");
    if (m < 1) return fail(TQ_EINVAL, "calibration needs at least one vector");
    if (!X_dev) return fail(TQ_EINVAL, "NULL device pointer");
    tq_status st = index_device_init(idx);
    if (st != TQ_OK) return st;
    const float *R = nullptr;
    st = rotation_dev(&idx->rot, &R);
    if (st != TQ_OK) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int d = idx->d;
    const size_t wb = (calib_workspace_bytes(d) + 255) & ~(size_t)255;
    AsyncBuf ws;
    hipError_t e = ws.alloc(wb + 2 * sizeof(float) * d, s);
    if (e != hipSuccess) return hip_fail(e, "hipMallocAsync(calibration workspace)");
    float *mu_d = reinterpret_cast<float *>(static_cast<uint8_t *>(ws.p) + wb);
    float *kappa_d = mu_d + d;
    e = hipMemsetAsync(idx->status, 0, sizeof(int), s);
    if (e == hipSuccess) e = calib_fit(X_dev, m, d, R, ws.p, idx->status, mu_d, kappa_d, s);
    if (e != hipSuccess) return hip_fail(e, "calibration");
    std::vector<float> mu((size_t)d), kappa((size_t)d);
    e = hipMemcpyAsync(mu.data(), mu_d, sizeof(float) * d, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipMemcpyAsync(kappa.data(), kappa_d, sizeof(float) * d, hipMemcpyDeviceToHost, s);
    if (e != hipSuccess) return hip_fail(e, "calibration read-back");
    int h = 0;
    st = read_status(idx->status, s, &h);   // synchronises the stream
    if (st != TQ_OK) return st;
    if (h & 1) return fail(TQ_EINVAL, "calibration batch has a zero or non-finite row");
    return install_calibration(idx, mu.data(), kappa.data());
}

tq_status tq_index_set_calibration(tq_index *idx, const float *mu_host, const float *kappa_host) {
    if (!idx || !mu_host || !kappa_host) return fail(TQ_EINVAL, "NULL argument");
    if (idx->n != 0) return fail(TQ_EINVAL, "calibration must precede the first vector");
    return install_calibration(idx, mu_host, kappa_host);
}

tq_status tq_index_calibration(const tq_index *idx, float *mu_host, float *kappa_host,
                               int32_t *calibrated) {
    if (!idx) return fail(TQ_EINVAL, "NULL index");
    if (calibrated) *calibrated = idx->calibrated ? 1 : 0;
    if (!idx->calibrated) return TQ_OK;
    if (mu_host) std::memcpy(mu_host, idx->mu_h.data(), sizeof(float) * idx->d);
    if (kappa_host) std::memcpy(kappa_host, idx->kappa_h.data(), sizeof(float) * idx->d);
    return TQ_OK;
}

}  // extern "C"

// New external ids must be valid, absent from the index and distinct.
static tq_status check_new_ids(const tq_index *x, const uint64_t *ids, int64_t n) {
    if (!ids) return fail(TQ_EINVAL, "NULL ids");
    std::unordered_map<uint64_t, int> seen;
    seen.reserve((size_t)n);
    for (int64_t i = 0; i < n; ++i) {
        if (ids[i] == UINT64_MAX) return fail(TQ_EINVAL, "id 2^64-1 is reserved");
        if (x->slot_of.count(ids[i])) return fail(TQ_EINVAL, "id already in the index");
        if (!seen.emplace(ids[i], 0).second) return fail(TQ_EINVAL, "repeated id in the batch");
    }
    return TQ_OK;
}

// Records the ids of the n slots from `base` on: external ids on the device,
// live bits, and the host map.
static tq_status commit_ids(tq_index *x, const uint64_t *ids, int64_t base, int64_t n,
                            hipStream_t s) {
    hipError_t e = hipMemcpyAsync(x->ext + base, ids, n * sizeof(uint64_t), hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = set_live(x->live, base, n, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(e, "id upload");
    for (int64_t i = 0; i < n; ++i) x->slot_of.emplace(ids[i], base + i);
    return TQ_OK;
}

static int64_t slot_lookup(const tq_index *x, uint64_t id) {
    if (!x->idmap) return id < (uint64_t)x->n ? (int64_t)id : -1;
    auto it = x->slot_of.find(id);
    return it == x->slot_of.end() ? -1 : it->second;
}

extern "C" {

tq_status tq_index_add_ids(tq_index *idx, const float *X_dev, const uint64_t *ids_host,
                           const uint16_t *tenants_dev, int64_t n, void *stream) {
    if (!idx) return fail(TQ_EINVAL, "NULL index");
    if (!idx->idmap) return fail(TQ_EINVAL, "not an id-map index");
    if (n < 0) return fail(TQ_EINVAL, "n < 0");
    if (n == 0) return TQ_OK;
    tq_status st = check_new_ids(idx, ids_host, n);
    if (st != TQ_OK) return st;
    const int64_t base = idx->n;
    st = add_vectors(idx, X_dev, tenants_dev, n, stream);
    if (st != TQ_OK) return st;
    return commit_ids(idx, ids_host, base, n, static_cast<hipStream_t>(stream));
}

tq_status tq_index_add_codes_ids(tq_index *idx, const uint8_t *codes_dev, const float *scales_dev,
                                 const uint64_t *ids_host, const uint16_t *tenants_dev, int64_t n,
                                 void *stream) {
    if (!idx) return fail(TQ_EINVAL, "NULL index");
    if (!idx->idmap) return fail(TQ_EINVAL, "not an id-map index");
    if (n < 0) return fail(TQ_EINVAL, "n < 0");
    if (n == 0) return TQ_OK;
    tq_status st = check_new_ids(idx, ids_host, n);
    if (st != TQ_OK) return st;
    const int64_t base = idx->n;
    st = add_codes_impl(idx, codes_dev, scales_dev, tenants_dev, n, stream);
    if (st != TQ_OK) return st;
    return commit_ids(idx, ids_host, base, n, static_cast<hipStream_t>(stream));
}

tq_status tq_index_remove_ids(tq_index *idx, const uint64_t *ids_host, int64_t n,
                              int64_t *removed_out) {
    if (!idx) return fail(TQ_EINVAL, "NULL index");
    if (!idx->idmap) return fail(TQ_EINVAL, "not an id-map index");
    if (n < 0 || (n > 0 && !ids_host)) return fail(TQ_EINVAL, "bad id list");
    std::unordered_map<int64_t, uint64_t> clear;   // block -> slots to retire
    int64_t removed = 0;
    for (int64_t i = 0; i < n; ++i) {
        auto it = idx->slot_of.find(ids_host[i]);
        if (it == idx->slot_of.end()) continue;
        const int64_t v = it->second;
        idx->slot_of.erase(it);
        clear[v >> 6] |= 1ull << (v & 63);
        ++removed;
    }
    if (removed > 0) {
        std::vector<int64_t> blocks;
        std::vector<uint64_t> masks;
        for (const auto &kv : clear) {
            blocks.push_back(kv.first);
            masks.push_back(kv.second);
        }
        DevBuf b, m;
        hipError_t e = b.alloc(blocks.size() * 8);
        if (e == hipSuccess) e = m.alloc(masks.size() * 8);
        if (e == hipSuccess) e = hipMemcpy(b.p, blocks.data(), blocks.size() * 8, hipMemcpyHostToDevice);
        if (e == hipSuccess) e = hipMemcpy(m.p, masks.data(), masks.size() * 8, hipMemcpyHostToDevice);
        if (e == hipSuccess)
            e = retire_slots(static_cast<const int64_t *>(b.p), static_cast<const uint64_t *>(m.p),
                             (int64_t)blocks.size(), idx->live, idx->tenants, idx->W, idx->summ, nullptr);
        if (e == hipSuccess) e = hipStreamSynchronize(nullptr);
        if (e != hipSuccess) return hip_fail(e, "deletion");
        idx->n_deleted += removed;
    }
    if (removed_out) *removed_out = removed;
    return TQ_OK;
}

tq_status tq_index_slots(const tq_index *idx, const uint64_t *ids_host, int64_t n,
                         int64_t *slots_host) {
    if (!idx) return fail(TQ_EINVAL, "NULL index");
    if (n < 0 || (n > 0 && (!ids_host || !slots_host))) return fail(TQ_EINVAL, "bad id list");
    for (int64_t i = 0; i < n; ++i) slots_host[i] = slot_lookup(idx, ids_host[i]);
    return TQ_OK;
}

tq_status tq_slot_allowlist(const tq_index *idx, const uint64_t *ids_host,
                            const int64_t *offsets_host, int64_t nq, uint64_t *bitmap_dev,
                            void *stream) {
    if (!idx) return fail(TQ_EINVAL, "NULL index");
    if (nq < 0 || (nq > 0 && (!offsets_host || !bitmap_dev))) return fail(TQ_EINVAL, "bad arguments");
    if (nq == 0) return TQ_OK;
    if (offsets_host[0] != 0) return fail(TQ_EINVAL, "offsets must start at 0");
    for (int64_t q = 0; q < nq; ++q)
        if (offsets_host[q + 1] < offsets_host[q]) return fail(TQ_EINVAL, "offsets must not decrease");
    if (offsets_host[nq] > 0 && !ids_host) return fail(TQ_EINVAL, "NULL ids");
    const int64_t nblk = (idx->n + 63) / 64;
    std::vector<uint64_t> bm((size_t)(nq * nblk), 0);
    for (int64_t q = 0; q < nq; ++q)
        for (int64_t j = offsets_host[q]; j < offsets_host[q + 1]; ++j) {
            const int64_t v = slot_lookup(idx, ids_host[j]);
            if (v >= 0) bm[(size_t)(q * nblk + (v >> 6))] |= 1ull << (v & 63);
        }
    if (bm.empty()) return TQ_OK;
    tq_status st = device_ready();
    if (st != TQ_OK) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e = hipMemcpyAsync(bitmap_dev, bm.data(), bm.size() * 8, hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(e, "allowlist upload");
    return TQ_OK;
}

tq_status tq_index_size(const tq_index *idx, int64_t *n_out) {
    if (!idx || !n_out) return fail(TQ_EINVAL, "NULL argument");
    *n_out = idx->n - idx->n_deleted;
    return TQ_OK;
}

tq_status tq_index_export(const tq_index *idx, uint8_t *codes_dev, float *scales_dev,
                          uint16_t *tenants_dev, void *stream) {
    if (!idx) return fail(TQ_EINVAL, "NULL index");
    if (idx->n == 0) return TQ_OK;
    tq_status st = device_ready();
    if (st != TQ_OK) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (codes_dev || scales_dev) {
        hipError_t e = blocked_to_canonical(idx->codes, idx->scales, idx->n, idx->d, idx->bits,
                                            codes_dev, scales_dev, s);
        if (e != hipSuccess) return hip_fail(e, "blocked_to_canonical");
    }
    if (tenants_dev) {
        hipError_t e = hipMemcpyAsync(tenants_dev, idx->tenants, idx->n * sizeof(uint16_t),
                                      hipMemcpyDeviceToDevice, s);
        if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync(tenants)");
    }
    return TQ_OK;
}

tq_status tq_index_info(const tq_index *idx, int32_t *d, int32_t *bits, int32_t *n_tenants,
                        int64_t *n, int32_t *idmap) {
    if (!idx) return fail(TQ_EINVAL, "NULL index");
    if (d) *d = idx->d;
    if (bits) *bits = idx->bits;
    if (n_tenants) *n_tenants = idx->T;
    if (n) *n = idx->n;
    if (idmap) *idmap = idx->idmap ? 1 : 0;
    return TQ_OK;
}

}  // extern "C"

namespace {

// ------------------------------------------------------------ persistence
// File layout (little-endian): FileHeader, then the canonical codes
// [n][d*bits/8], the scales [n] float32 and the tenant ids [n] uint16; for
// an id-map index (flag 1) the external ids [n] uint64 and the live-slot
// masks [ceil(n/64)] uint64; for a TQ+ calibrated index (flag 2) mu [d] and
// kappa [d] float32; then a 64-bit FNV-1a hash of every preceding byte.
constexpr char kFileMagic[8] = {'T', 'Q', 'I', 'N', 'D', 'E', 'X', '1'};
constexpr uint32_t kFileVersion = 1;
constexpr uint32_t kFileIds = 1;
constexpr uint32_t kFileCalib = 2;

struct FileHeader {
    char magic[8];
    uint32_t version;
    uint32_t flags;          // kFileIds / kFileCalib: optional sections present
    int32_t d, bits;
    uint64_t seed;           // rotation seed
    int64_t n;
    int32_t n_tenants;
    int32_t reserved;
};
static_assert(sizeof(FileHeader) == 48, "file header layout");

struct Fnv1a {
    uint64_t h = 1469598103934665603ull;
    void add(const void *p, size_t n) {
        const uint8_t *b = static_cast<const uint8_t *>(p);
        for (size_t i = 0; i < n; ++i) h = (h ^ b[i]) * 1099511628211ull;
    }
};

struct FileCloser {
    FILE *f;
    ~FileCloser() {
        if (f) fclose(f);
    }
};

}  // namespace

extern "C" {

tq_status tq_index_save(const tq_index *idx, const char *path) {
    if (!idx || !path) return fail(TQ_EINVAL, "NULL argument");
    const int64_t n = idx->n;
    const size_t cbytes = (size_t)idx->d * idx->bits / 8;
    std::vector<uint8_t> codes((size_t)n * cbytes);
    std::vector<float> scales((size_t)n);
    std::vector<uint16_t> ten((size_t)n);
    const int64_t nb = (n + 63) / 64;
    std::vector<uint64_t> ext(idx->idmap ? (size_t)n : 0), live(idx->idmap ? (size_t)nb : 0);
    if (n > 0) {
        tq_status st = device_ready();
        if (st != TQ_OK) return st;
        DevBuf c, sc, t;
        hipError_t e = c.alloc(codes.size());
        if (e == hipSuccess) e = sc.alloc(scales.size() * 4);
        if (e == hipSuccess) e = t.alloc(ten.size() * 2);
        if (e != hipSuccess) return hip_fail(e, "hipMalloc(save staging)");
        st = tq_index_export(idx, static_cast<uint8_t *>(c.p), static_cast<float *>(sc.p),
                             static_cast<uint16_t *>(t.p), nullptr);
        if (st != TQ_OK) return st;
        e = hipMemcpy(codes.data(), c.p, codes.size(), hipMemcpyDeviceToHost);
        if (e == hipSuccess) e = hipMemcpy(scales.data(), sc.p, scales.size() * 4, hipMemcpyDeviceToHost);
        if (e == hipSuccess) e = hipMemcpy(ten.data(), t.p, ten.size() * 2, hipMemcpyDeviceToHost);
        if (e == hipSuccess && idx->idmap)
            e = hipMemcpy(ext.data(), idx->ext, ext.size() * 8, hipMemcpyDeviceToHost);
        if (e == hipSuccess && idx->idmap)
            e = hipMemcpy(live.data(), idx->live, live.size() * 8, hipMemcpyDeviceToHost);
        if (e != hipSuccess) return hip_fail(e, "index read-back");
    }
    FileHeader h{};
    std::memcpy(h.magic, kFileMagic, 8);
    h.version = kFileVersion;
    h.flags = (idx->idmap ? kFileIds : 0) | (idx->calibrated ? kFileCalib : 0);
    h.d = idx->d;
    h.bits = idx->bits;
    h.seed = idx->rot.seed;
    h.n = n;
    h.n_tenants = idx->T;
    FileCloser fc{fopen(path, "wb")};
    if (!fc.f) return fail(TQ_EINVAL, std::string("cannot open ") + path + " for writing");
    Fnv1a fnv;
    bool ok = true;
    auto put = [&](const void *p, size_t bytes) {
        if (ok && bytes && fwrite(p, 1, bytes, fc.f) != bytes) ok = false;
        fnv.add(p, bytes);
    };
    put(&h, sizeof h);
    put(codes.data(), codes.size());
    put(scales.data(), scales.size() * 4);
    put(ten.data(), ten.size() * 2);
    put(ext.data(), ext.size() * 8);
    put(live.data(), live.size() * 8);
    if (idx->calibrated) {
        put(idx->mu_h.data(), idx->mu_h.size() * 4);
        put(idx->kappa_h.data(), idx->kappa_h.size() * 4);
    }
    const uint64_t sum = fnv.h;
    if (ok && fwrite(&sum, 1, 8, fc.f) != 8) ok = false;
    const int rc = fclose(fc.f);
    fc.f = nullptr;
    if (!ok || rc != 0) return fail(TQ_EINVAL, std::string("write to ") + path + " failed");
    return TQ_OK;
}

tq_status tq_index_load(const char *path, const tq_codebook *cb, const tq_rotation *rot,
                        tq_index **out) {
    if (!out) return fail(TQ_EINVAL, "out is NULL");
    *out = nullptr;
    if (!path || !cb || !rot) return fail(TQ_EINVAL, "NULL argument");
    FileCloser fc{fopen(path, "rb")};
    if (!fc.f) return fail(TQ_EINVAL, std::string("cannot open ") + path);
    Fnv1a fnv;
    bool ok = true;
    auto get = [&](void *p, size_t bytes) {
        if (ok && bytes && fread(p, 1, bytes, fc.f) != bytes) ok = false;
        if (ok) fnv.add(p, bytes);
    };
    FileHeader h{};
    get(&h, sizeof h);
    if (!ok || std::memcmp(h.magic, kFileMagic, 8) != 0)
        return fail(TQ_EINVAL, std::string(path) + " is not an index file");
    if (h.version != kFileVersion || (h.flags & ~(kFileIds | kFileCalib)) != 0)
        return fail(TQ_EUNSUPPORTED, "index file version or sections not supported");
    const bool ids = (h.flags & kFileIds) != 0;
    const bool calib = (h.flags & kFileCalib) != 0;
    if (h.d != cb->t.d || h.bits != cb->t.bits)
        return fail(TQ_EINVAL, "index file d/bits differ from the codebook's");
    if (h.d != rot->d || h.seed != rot->seed)
        return fail(TQ_EINVAL, "index file d/seed differ from the rotation's");
    if (h.n < 0 || h.n > (int64_t)INT32_MAX || h.n_tenants < 1 || h.n_tenants > 65535)
        return fail(TQ_EINVAL, "index file header out of range");
    const int64_t n = h.n;
    const size_t cbytes = (size_t)h.d * h.bits / 8;
    const int64_t nb = (n + 63) / 64;
    std::vector<uint8_t> codes;
    std::vector<float> scales;
    std::vector<uint16_t> ten;
    std::vector<uint64_t> ext, live;
    std::vector<float> mu, kappa;
    try {
        if (calib) {
            mu.resize((size_t)h.d);
            kappa.resize((size_t)h.d);
        }
        codes.resize((size_t)n * cbytes);
        scales.resize((size_t)n);
        ten.resize((size_t)n);
        if (ids) {
            ext.resize((size_t)n);
            live.resize((size_t)nb);
        }
    } catch (const std::bad_alloc &) {
        return fail(TQ_ENOMEM, "host allocation failed");
    }
    get(codes.data(), codes.size());
    get(scales.data(), scales.size() * 4);
    get(ten.data(), ten.size() * 2);
    get(ext.data(), ext.size() * 8);
    get(live.data(), live.size() * 8);
    get(mu.data(), mu.size() * 4);
    get(kappa.data(), kappa.size() * 4);
    uint64_t sum = 0;
    if (!ok || fread(&sum, 1, 8, fc.f) != 8) return fail(TQ_EINVAL, std::string(path) + " is truncated");
    if (sum != fnv.h) return fail(TQ_EINVAL, std::string(path) + " fails its checksum");
    if (fgetc(fc.f) != EOF) return fail(TQ_EINVAL, std::string(path) + " has trailing bytes");
    // the id sections: live bits only on existing slots, live ids distinct
    std::unordered_map<uint64_t, int64_t> slot_of;
    int64_t n_live = 0;
    if (ids) {
        for (int64_t b = 0; b < nb; ++b) {
            const int valid = (int)std::min<int64_t>(64, n - b * 64);
            if (valid < 64 && (live[(size_t)b] >> valid) != 0)
                return fail(TQ_EINVAL, std::string(path) + ": live bit on a missing slot");
        }
        slot_of.reserve((size_t)n);
        for (int64_t v = 0; v < n; ++v) {
            if (!((live[(size_t)(v >> 6)] >> (v & 63)) & 1ull)) continue;
            if (ext[(size_t)v] == UINT64_MAX || !slot_of.emplace(ext[(size_t)v], v).second)
                return fail(TQ_EINVAL, std::string(path) + ": invalid or repeated live id");
            ++n_live;
        }
    }
    tq_index *x = nullptr;
    tq_status st = ids ? tq_idmap_create(cb, rot, h.n_tenants, &x)
                       : tq_index_create(cb, rot, h.n_tenants, &x);
    if (st != TQ_OK) return st;
    if (calib) {
        st = install_calibration(x, mu.data(), kappa.data());
        if (st != TQ_OK) {
            tq_index_free(x);
            return st;
        }
    }
    if (n > 0) {
        st = index_grow(x, n, nullptr);
        DevBuf c, sc, t;
        hipError_t e = hipSuccess;
        if (st == TQ_OK) {
            e = c.alloc(codes.size());
            if (e == hipSuccess) e = sc.alloc(scales.size() * 4);
            if (e == hipSuccess) e = t.alloc(ten.size() * 2);
            if (e == hipSuccess) e = hipMemcpy(c.p, codes.data(), codes.size(), hipMemcpyHostToDevice);
            if (e == hipSuccess) e = hipMemcpy(sc.p, scales.data(), scales.size() * 4, hipMemcpyHostToDevice);
            if (e == hipSuccess) e = hipMemcpy(t.p, ten.data(), ten.size() * 2, hipMemcpyHostToDevice);
            st = e != hipSuccess ? hip_fail(e, "index upload")
                                 : add_codes_impl(x, static_cast<const uint8_t *>(c.p),
                                                  static_cast<const float *>(sc.p),
                                                  static_cast<const uint16_t *>(t.p), n, nullptr);
        }
        if (st == TQ_OK && ids) {
            // ids and live masks as saved; blocks with dead slots get their
            // summaries rebuilt over the live ones
            hipError_t e = hipMemcpy(x->ext, ext.data(), ext.size() * 8, hipMemcpyHostToDevice);
            if (e == hipSuccess) e = hipMemcpy(x->live, live.data(), live.size() * 8, hipMemcpyHostToDevice);
            std::vector<int64_t> blocks;
            for (int64_t b = 0; b < nb; ++b) {
                const int valid = (int)std::min<int64_t>(64, n - b * 64);
                const uint64_t full = valid == 64 ? ~0ull : ((1ull << valid) - 1);
                if (live[(size_t)b] != full) blocks.push_back(b);
            }
            if (e == hipSuccess && !blocks.empty()) {
                std::vector<uint64_t> zero(blocks.size(), 0);
                DevBuf bb, zz;
                e = bb.alloc(blocks.size() * 8);
                if (e == hipSuccess) e = zz.alloc(zero.size() * 8);
                if (e == hipSuccess) e = hipMemcpy(bb.p, blocks.data(), blocks.size() * 8, hipMemcpyHostToDevice);
                if (e == hipSuccess) e = hipMemcpy(zz.p, zero.data(), zero.size() * 8, hipMemcpyHostToDevice);
                if (e == hipSuccess)
                    e = retire_slots(static_cast<const int64_t *>(bb.p), static_cast<const uint64_t *>(zz.p),
                                     (int64_t)blocks.size(), x->live, x->tenants, x->W, x->summ, nullptr);
                if (e == hipSuccess) e = hipStreamSynchronize(nullptr);
            }
            if (e != hipSuccess) st = hip_fail(e, "id upload");
            x->slot_of.swap(slot_of);
            x->n_deleted = n - n_live;
        }
        if (st != TQ_OK) {
            tq_index_free(x);
            return st;
        }
    }
    *out = x;
    return TQ_OK;
}

void tq_index_free(tq_index *idx) {
    if (!idx) return;
    index_release(idx);
    if (idx->rot.R_dev) (void)hipFree(idx->rot.R_dev);
    idx->rot.R_dev = nullptr;
    delete idx;
}

static ScanShape shape_of(const tq_index *x) {
    ScanShape s;
    s.d = x->d;
    s.bits = x->bits;
    s.chunks = x->chunks;
    s.n = x->n;
    s.nblk = (x->n + 63) / 64;
    s.W = x->W;
    return s;
}

// Workgroups of the search kernels: one per compute unit, or TQ_SCAN_GRID
// (1..65535) when set, which gives each workgroup a larger share of the
// blocks (at one workgroup, a 300K-row index spans several list windows of
// the filtered scan).
static int scan_grid() {
    if (const char *e = getenv("TQ_SCAN_GRID")) {
        char *end = nullptr;
        const long v = strtol(e, &end, 10);
        if (end != e && *end == '\0' && v >= 1 && v <= 65535) return (int)v;
    }
    const int cus = device_cu_count();
    return cus > 0 ? cus : 256;
}

static bool use_mfma(const ScanShape &sh, int k, int base) {
    return base == TQ_PATH_MFMA && mfma_search_supported(sh, k);
}

// Workspace of a search; a calibrated index adds the queries' constant
// terms at the end (calib_offset).
static size_t calib_offset(const ScanShape &sh, int64_t nq, int k) {
    return (lut_search_workspace_bytes(sh, nq, k, scan_grid()) + 255) & ~(size_t)255;
}

static size_t search_bytes(const ScanShape &sh, int64_t nq, int k, int base, bool calibrated) {
    if (use_mfma(sh, k, base)) return mfma_search_workspace_bytes(sh, nq, k, scan_grid());
    if (calibrated) return calib_offset(sh, nq, k) + (size_t)nq * sizeof(float);
    return lut_search_workspace_bytes(sh, nq, k, scan_grid());
}

// With TQ+ calibration the scans take kappa * q' (written over the rotated
// queries at the start of the workspace) and the constant terms.
static tq_status prepare_calibrated(const tq_index *x, const float *Qrot, int64_t nq, float *qout,
                                    float *qconst, hipStream_t s) {
    hipError_t e = calib_queries(Qrot, nq, x->d, x->mu, x->kappa, qout, qconst, s);
    if (e != hipSuccess) return hip_fail(e, "query calibration");
    return TQ_OK;
}

// max |float16(c)| and max |float16(c) - c| over the float32 centroids
static void centroid_half_bounds(const tq_index *x, float *cmax16, float *dmax) {
    float m = 0.f, dm = 0.f;
    for (int i = 0; i < (1 << x->bits); ++i) {
        const float c = x->cbdev.cents32[i];
        const float h = (float)(_Float16)c;
        m = std::max(m, std::fabs(h));
        dm = std::max(dm, std::fabs(h - c));
    }
    *cmax16 = m;
    *dmax = dm;
}

tq_status tq_search_workspace_size(const tq_index *idx, int64_t nq, int32_t k, int32_t path,
                                   size_t *bytes_out) {
    if (!idx || !bytes_out) return fail(TQ_EINVAL, "NULL argument");
    if (nq < 0) return fail(TQ_EINVAL, "nq < 0");
    if (k < 1 || k > kMaxK) return fail(TQ_EINVAL, "k must be in 1..4096");
    const int base = path & ~(TQ_FLAG_PREROTATED | TQ_FLAG_SLOT_ALLOW);
    if (base != TQ_PATH_AUTO && base != TQ_PATH_LUT && base != TQ_PATH_MFMA)
        return fail(TQ_EINVAL, "unknown path");
    if (base == TQ_PATH_MFMA && !mfma_search_supported(shape_of(idx), k))
        return fail(TQ_EUNSUPPORTED, "matrix-core path needs 4-bit codes, d % 256 == 0, d <= 1792, "
                                     "k <= 256 and at most 4096 tenants");
    if (base == TQ_PATH_MFMA && idx->calibrated)
        return fail(TQ_EUNSUPPORTED, "matrix-core path does not take a TQ+ calibrated index");
    tq_status st = device_ready();
    if (st != TQ_OK) return st;
    *bytes_out = search_bytes(shape_of(idx), nq, k, base, idx->calibrated);
    return TQ_OK;
}

tq_status tq_search_ex(const tq_index *idx, const float *Q_dev, int64_t nq, int32_t k,
                       const uint64_t *allow_dev, int32_t path, void *workspace_dev,
                       size_t workspace_bytes, int64_t *ids_dev, float *scores_dev,
                       void *stream) {
    if (!idx) return fail(TQ_EINVAL, "NULL index");
    if (nq < 0) return fail(TQ_EINVAL, "nq < 0");
    if (k < 1 || k > kMaxK) return fail(TQ_EINVAL, "k must be in 1..4096");
    const bool prerotated = (path & TQ_FLAG_PREROTATED) != 0;
    const bool slot_allow = (path & TQ_FLAG_SLOT_ALLOW) != 0;
    const int base = path & ~(TQ_FLAG_PREROTATED | TQ_FLAG_SLOT_ALLOW);
    if (base != TQ_PATH_AUTO && base != TQ_PATH_LUT && base != TQ_PATH_MFMA)
        return fail(TQ_EINVAL, "unknown path");
    if (nq == 0) return TQ_OK;
    if (!Q_dev || !ids_dev || !scores_dev) return fail(TQ_EINVAL, "NULL device pointer");
    if (!workspace_dev) return fail(TQ_EINVAL, "NULL workspace");
    if (((uintptr_t)workspace_dev & 255) != 0) return fail(TQ_EINVAL, "workspace must be 256-byte aligned");
    tq_status st = device_ready();
    if (st != TQ_OK) return st;
    const ScanShape sh = shape_of(idx);
    if (base == TQ_PATH_MFMA && !mfma_search_supported(sh, k))
        return fail(TQ_EUNSUPPORTED, "matrix-core path needs 4-bit codes, d % 256 == 0, d <= 1792, "
                                     "k <= 256 and at most 4096 tenants");
    if (slot_allow && !allow_dev) return fail(TQ_EINVAL, "slot allowlist flag without an allowlist");
    SearchFilter filter;
    if (slot_allow)
        filter.slot_allow = allow_dev;
    else
        filter.allow = allow_dev;
    if (idx->idmap && idx->n_deleted > 0) filter.live = idx->live;
    if (base == TQ_PATH_MFMA && (filter.live || filter.slot_allow))
        return fail(TQ_EUNSUPPORTED, "matrix-core path takes tenant allowlists only "
                                     "(no deleted slots, no slot allowlists)");
    if (base == TQ_PATH_MFMA && idx->calibrated)
        return fail(TQ_EUNSUPPORTED, "matrix-core path does not take a TQ+ calibrated index");
    const int grid = scan_grid();
    const size_t need = search_bytes(sh, nq, k, base, idx->calibrated);
    if (workspace_bytes < need)
        return fail(TQ_EINVAL, "workspace too small: need " + std::to_string(need) + " bytes");
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (idx->n == 0) {
        // nothing indexed: every slot is padding
        std::vector<int64_t> pad_i((size_t)nq * k, -1);
        std::vector<float> pad_s((size_t)nq * k, -INFINITY);
        hipError_t e = hipMemcpyAsync(ids_dev, pad_i.data(), pad_i.size() * 8, hipMemcpyHostToDevice, s);
        if (e == hipSuccess)
            e = hipMemcpyAsync(scores_dev, pad_s.data(), pad_s.size() * 4, hipMemcpyHostToDevice, s);
        if (e == hipSuccess) e = hipStreamSynchronize(s);
        if (e != hipSuccess) return hip_fail(e, "padding copy");
        return TQ_OK;
    }
    // the LUT path's global bounds are set by the query rotation's launch:
    // the scan then follows the rotation with no launch in between
    bool bounds_ready = false;
    const float *Qrot = Q_dev;
    if (!prerotated) {
        const float *R = nullptr;
        st = rotation_dev(&idx->rot, &R);
        if (st != TQ_OK) return st;
        float *qr = static_cast<float *>(workspace_dev);
        int *bounds = use_mfma(sh, k, base) ? nullptr
                                            : lut_search_bounds(sh, nq, k, grid, workspace_dev);
        hipError_t e = rotate_rows_f32(Q_dev, nq, idx->d, R, qr, s, bounds, bounds ? nq : 0,
                                       kBoundInit);
        if (e != hipSuccess) return hip_fail(e, "query rotation");
        bounds_ready = bounds != nullptr;
        Qrot = qr;
    }
    float *qconst = nullptr;
    if (idx->calibrated) {
        uint8_t *w8 = static_cast<uint8_t *>(workspace_dev);
        qconst = reinterpret_cast<float *>(w8 + calib_offset(sh, nq, k));
        float *qr = static_cast<float *>(workspace_dev);
        st = prepare_calibrated(idx, Qrot, nq, qr, qconst, s);
        if (st != TQ_OK) return st;
        Qrot = qr;
    }
    if (use_mfma(sh, k, base)) {
        int n_fallback = 0;
        float cmax16 = 0.f, dmax = 0.f;
        centroid_half_bounds(idx, &cmax16, &dmax);
        hipError_t e = mfma_search(sh, idx->codes, idx->scales, scale_max_dev(idx), idx->tenants,
                                   idx->summ, idx->cents_dev, cmax16, dmax, Qrot, nq, k,
                                   allow_dev, grid, workspace_dev, ids_dev, scores_dev,
                                   &n_fallback, s);
        if (e != hipSuccess) return hip_fail(e, "matrix-core search");
        if (idx->idmap && (e = map_ids(ids_dev, nq * k, idx->ext, s)) != hipSuccess)
            return hip_fail(e, "id mapping");
        g_last_fallbacks = n_fallback;
        return TQ_OK;
    }
    hipError_t e = lut_search(sh, idx->codes, idx->scales, idx->tenants, idx->summ, idx->cents_dev,
                              Qrot, nq, k, filter, grid, workspace_dev, workspace_bytes, ids_dev,
                              scores_dev, s, qconst, bounds_ready);
    if (e != hipSuccess) return hip_fail(e, "scan");
    if (idx->idmap && (e = map_ids(ids_dev, nq * k, idx->ext, s)) != hipSuccess)
        return hip_fail(e, "id mapping");
    g_last_fallbacks = 0;
    return TQ_OK;
}

tq_status tq_search_postfilter(const tq_index *idx, const float *Q_dev, int64_t nq, int32_t k,
                               int32_t overfetch, const uint64_t *allow_dev, int64_t *ids_dev,
                               float *scores_dev, void *stream) {
    if (!idx) return fail(TQ_EINVAL, "NULL index");
    if (nq < 0) return fail(TQ_EINVAL, "nq < 0");
    if (k < 1 || overfetch < 1) return fail(TQ_EINVAL, "k and overfetch must be positive");
    if ((int64_t)k * overfetch > kMaxK) return fail(TQ_EUNSUPPORTED, "k * overfetch must be <= 4096");
    if (nq == 0) return TQ_OK;
    if (!Q_dev || !allow_dev || !ids_dev || !scores_dev) return fail(TQ_EINVAL, "NULL device pointer");
    tq_status st = device_ready();
    if (st != TQ_OK) return st;
    const int kk = k * overfetch;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (idx->n == 0) {
        // nothing indexed: every slot is padding
        std::vector<int64_t> pad_i((size_t)nq * k, -1);
        std::vector<float> pad_s((size_t)nq * k, -INFINITY);
        hipError_t e = hipMemcpyAsync(ids_dev, pad_i.data(), pad_i.size() * 8, hipMemcpyHostToDevice, s);
        if (e == hipSuccess)
            e = hipMemcpyAsync(scores_dev, pad_s.data(), pad_s.size() * 4, hipMemcpyHostToDevice, s);
        if (e == hipSuccess) e = hipStreamSynchronize(s);
        if (e != hipSuccess) return hip_fail(e, "padding copy");
        return TQ_OK;
    }
    const ScanShape sh = shape_of(idx);
    const int grid = scan_grid();
    const size_t sbytes =
        (search_bytes(sh, nq, kk, TQ_PATH_LUT, idx->calibrated) + 255) & ~(size_t)255;
    const size_t tbytes = (size_t)nq * kk * (sizeof(int64_t) + sizeof(float));
    AsyncBuf ws;
    hipError_t e = ws.alloc(sbytes + tbytes, s);
    if (e != hipSuccess) return hip_fail(e, "hipMallocAsync(post-filter workspace)");
    uint8_t *w8 = static_cast<uint8_t *>(ws.p);
    int64_t *ids_tmp = reinterpret_cast<int64_t *>(w8 + sbytes);
    float *sc_tmp = reinterpret_cast<float *>(ids_tmp + (size_t)nq * kk);
    const float *R = nullptr;
    st = rotation_dev(&idx->rot, &R);
    if (st != TQ_OK) return st;
    float *qr = reinterpret_cast<float *>(w8);
    e = rotate_rows_f32(Q_dev, nq, idx->d, R, qr, s);
    if (e != hipSuccess) return hip_fail(e, "query rotation");
    float *qconst = nullptr;
    if (idx->calibrated) {
        qconst = reinterpret_cast<float *>(w8 + calib_offset(sh, nq, kk));
        st = prepare_calibrated(idx, qr, nq, qr, qconst, s);
        if (st != TQ_OK) return st;
    }
    // the unfiltered top k * overfetch (deleted vectors excluded) ...
    SearchFilter f;
    if (idx->idmap && idx->n_deleted > 0) f.live = idx->live;
    e = lut_search(sh, idx->codes, idx->scales, idx->tenants, idx->summ, idx->cents_dev, qr, nq, kk,
                   f, grid, w8, sbytes, ids_tmp, sc_tmp, s, qconst);
    if (e != hipSuccess) return hip_fail(e, "scan");
    // ... then the first k whose tenant is allowed
    e = postfilter(ids_tmp, sc_tmp, nq, kk, idx->tenants, allow_dev, idx->W, k, ids_dev, scores_dev, s);
    if (e == hipSuccess && idx->idmap) e = map_ids(ids_dev, nq * k, idx->ext, s);
    if (e != hipSuccess) return hip_fail(e, "post-filter");
    g_last_fallbacks = 0;
    return TQ_OK;
}

tq_status tq_search(const tq_index *idx, const float *Q_dev, int64_t nq, int32_t k,
                    const uint64_t *allow_dev, int64_t *ids_dev, float *scores_dev, void *stream) {
    size_t bytes = 0;
    tq_status st = tq_search_workspace_size(idx, nq, k, TQ_PATH_AUTO, &bytes);
    if (st != TQ_OK) return st;
    if (nq == 0) return TQ_OK;
    hipStream_t s = static_cast<hipStream_t>(stream);
    AsyncBuf ws;
    hipError_t e = ws.alloc(bytes, s);
    if (e != hipSuccess) return hip_fail(e, "hipMallocAsync(search workspace)");
    return tq_search_ex(idx, Q_dev, nq, k, allow_dev, TQ_PATH_AUTO, ws.p, bytes, ids_dev,
                        scores_dev, stream);
}

}  // extern "C"
