// Rotation + quantisation of float32 rows on gfx950 (section II-B, steps 1-5).
//
// Pipeline per chunk of rows:
//  1. rot_gemm<QuantEpilogue>: Y = X R^T on the matrix cores
//     (v_mfma_f32_16x16x4_f32), with each 32-wide slab of k accumulated in
//     float32 and then added into float64 accumulators.  The same kernel
//     computes the exact row norm n = sqrt(sum_k x_k^2) (sequential float64
//     over k, from the staged A tile) and reports non-finite inputs.  The
//     epilogue turns every y into a code by comparing it with fl64(t_i * n)
//     and flags the coordinate when y lies within tau of a threshold, where
//     tau bounds |y - S| for S the float64 sequential dot product of the
//     definition:
//       per slab, float32 MFMA accumulation of 32 products from 0:
//         |err| <= gamma_33 * sum|R_jk x_k|   (gamma_m = m u / (1 - m u),
//                                              u = 2^-24; doubled for margin)
//       float64 sum of 48 slab partials and the float64 reference itself:
//         < 2e-13 * n;  flushed denormal products: < 2e-35 absolute.
//     With ||R_j|| <= 1 + 1e-6 this gives tau = 4.0e-6 * n + 1e-30.
//  2. fixup: every flagged coordinate is recomputed as the sequential float64
//     sum sum_{k=0}^{d-1} R[j][k] x_k (every product of two float32 values is
//     exact in float64) and re-coded.  Flags are kept per output tile; with
//     few flags per tile (b <= 4) one thread per flag reads its rows from
//     memory, with many (b = 8, about 2% of coordinates) each tile stages
//     its X and R slabs in LDS once for all of its flags.
//  3. pack: per row, scale = n / sqrt(sum_j fl64(c_code_j^2)) (sequential
//     float64 over j) and the codes are written in the canonical bitstream
//     and/or the index's blocked layout.
// With TQ+ calibration (section II-B) coordinate j is coded against its own
// thresholds fl64(a_ij n), a_ij = fl64(mu_j + fl64(kappa_j t_i)), and the
// scale uses yhat_j = fl64(mu_j + fl64(kappa_j c_code_j)); both tables are
// computed on the host in float64 and passed in (CalibDev).
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "kernels.h"

namespace tq {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int BM = 128;                 // rows of X per workgroup
constexpr int BN = 128;                 // rows of R (output columns) per workgroup
constexpr int KB = 32;                  // k per slab
constexpr int LDS_STRIDE = KB + 4;      // floats per staged row (conflict-free b128 reads)
constexpr int GEMM_THREADS = 512;       // 8 waves: 2 along rows x 4 along columns
constexpr double kTauRel = 4.0e-6;
constexpr double kTauAbs = 1e-30;

struct QuantArgs {
    const double *bounds;   // device copy of the thresholds t_i (levels-1)
    // TQ+ calibration: per-coordinate thresholds a_ij = mu_j + kappa_j t_i,
    // [levels-1][d] (null: the shared t_i)
    const double *athr;
    int levels;
    uint8_t *codes_tmp;     // [rows][d] unpacked codes of this chunk
    double *norms;          // [rows] exact row norms (written by column tile 0)
    uint32_t *flags;        // per output tile, BM * BN slots: flagged (local row << 7 | local col)
    unsigned int *tile_count;   // flags of each output tile
    int *status;            // set non-zero on a non-finite input
};

struct F32Args {
    float *Y;               // [rows][d]
};

// XCD-aware tile order: the d/BN column tiles of one row tile go to the same
// XCD (workgroups are dealt to the 8 XCDs round-robin), so the X tile is read
// from HBM once and then served by that XCD's L2.
__device__ inline void tile_of(int bid, int ncol, int &rt, int &ct) {
    const int x = bid & 7;
    const int rest = bid >> 3;
    ct = rest % ncol;
    rt = (rest / ncol) * 8 + x;
}

template <bool QUANT>
__global__ __launch_bounds__(GEMM_THREADS) void rot_gemm(
    const float *__restrict__ X, int64_t m, const float *__restrict__ R, int d,
    int n_row_tiles, QuantArgs qa, F32Args fa) {
    __shared__ __attribute__((aligned(16))) float As[2][BM * LDS_STRIDE];
    __shared__ __attribute__((aligned(16))) float Bs[2][BN * LDS_STRIDE];
    __shared__ double norm_s[BM];
    __shared__ double bnd_s[255];   // the shared thresholds t_i (no TQ+ tables)
    // TQ+ thresholds of this tile's columns, [levels-1][BN], for b <= 4
    __shared__ double athr_s[QUANT ? 15 * BN : 1];
    __shared__ unsigned int nflag_s;

    const int ncol = (d + BN - 1) / BN;
    int rt, ct;
    tile_of(blockIdx.x, ncol, rt, ct);
    if (rt >= n_row_tiles) return;
    const int64_t row0 = (int64_t)rt * BM;
    const int col0 = ct * BN;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wr = wave >> 2;     // 0..1 : 64-row half
    const int wc = wave & 3;      // 0..3 : 32-column quarter
    const int l16 = lane & 15;
    const int g4 = lane >> 4;

    // global -> register prefetch: 2 float4 of A and 2 of B per thread per slab
    f4 pa[2], pb[2];
    auto load_slab = [&](int k0) {
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            const int e = tid + r * GEMM_THREADS;
            const int row = e >> 3;
            const int kq = (e & 7) * 4;
            const int64_t gr = row0 + row;
            if (gr < m)
                pa[r] = *reinterpret_cast<const f4 *>(X + gr * d + k0 + kq);
            else
                pa[r] = f4{0.f, 0.f, 0.f, 0.f};
            if (col0 + row < d)
                pb[r] = *reinterpret_cast<const f4 *>(R + (int64_t)(col0 + row) * d + k0 + kq);
            else
                pb[r] = f4{0.f, 0.f, 0.f, 0.f};
        }
    };
    auto store_slab = [&](int buf) {
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            const int e = tid + r * GEMM_THREADS;
            const int row = e >> 3;
            const int kq = (e & 7) * 4;
            *reinterpret_cast<f4 *>(&As[buf][row * LDS_STRIDE + kq]) = pa[r];
            *reinterpret_cast<f4 *>(&Bs[buf][row * LDS_STRIDE + kq]) = pb[r];
        }
    };

    f4 acc[4][2];
    double accd[4][2][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int v = 0; v < 4; ++v) accd[i][j][v] = 0.0;
        }
    double nrm2 = 0.0;       // sequential sum of squares (threads < BM own a row)
    bool finite = true;

    const int nslab = d / KB;
    if (QUANT && !qa.athr)
        for (int i = tid; i < qa.levels - 1; i += GEMM_THREADS) bnd_s[i] = qa.bounds[i];
    const bool athr_lds = QUANT && qa.athr && qa.levels <= 16;
    if (athr_lds)
        for (int e = tid; e < (qa.levels - 1) * BN; e += GEMM_THREADS) {
            const int i = e / BN, c = col0 + e % BN;
            athr_s[e] = c < d ? qa.athr[(int64_t)i * d + c] : 0.0;
        }
    if (QUANT && tid == 0) nflag_s = 0;
    load_slab(0);
    store_slab(0);
    __syncthreads();
    for (int s = 0; s < nslab; ++s) {
        const int buf = s & 1;
        if (s + 1 < nslab) load_slab((s + 1) * KB);
        if (QUANT && tid < BM) {
            // row norm, k in order
            const float *a = &As[buf][tid * LDS_STRIDE];
#pragma unroll
            for (int q = 0; q < KB; q += 4) {
                const f4 v = *reinterpret_cast<const f4 *>(a + q);
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const double xv = (double)v[c];
                    finite = finite && std::isfinite(v[c]);
                    const double sq = xv * xv;
                    nrm2 = nrm2 + sq;
                }
            }
        }
#pragma unroll
        for (int sub = 0; sub < KB / 16; ++sub) {
            f4 af[4], bf[2];
#pragma unroll
            for (int ti = 0; ti < 4; ++ti)
                af[ti] = *reinterpret_cast<const f4 *>(
                    &As[buf][(wr * 64 + ti * 16 + l16) * LDS_STRIDE + sub * 16 + g4 * 4]);
#pragma unroll
            for (int tj = 0; tj < 2; ++tj)
                bf[tj] = *reinterpret_cast<const f4 *>(
                    &Bs[buf][(wc * 32 + tj * 16 + l16) * LDS_STRIDE + sub * 16 + g4 * 4]);
#pragma unroll
            for (int st = 0; st < 4; ++st)
#pragma unroll
                for (int ti = 0; ti < 4; ++ti)
#pragma unroll
                    for (int tj = 0; tj < 2; ++tj)
                        acc[ti][tj] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                            af[ti][st], bf[tj][st], acc[ti][tj], 0, 0, 0);
        }
        // fold the slab's float32 partials into float64
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j) {
#pragma unroll
                for (int v = 0; v < 4; ++v) accd[i][j][v] += (double)acc[i][j][v];
                acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};
            }
        if (s + 1 < nslab) store_slab(buf ^ 1);
        __syncthreads();
    }

    if (QUANT) {
        if (tid < BM) {
            const double nrm = std::sqrt(nrm2);
            norm_s[tid] = nrm;
            const int64_t gr = row0 + tid;
            if (gr < m) {
                if (ct == 0) qa.norms[gr] = nrm;
                if (!finite) atomicOr(qa.status, 1);
            }
        }
        __syncthreads();
        const int L = qa.levels;
        const int64_t tile = (int64_t)rt * ncol + ct;
        uint32_t *tflags = qa.flags + tile * (BM * BN);
#pragma unroll
        for (int ti = 0; ti < 4; ++ti)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int lr = wr * 64 + ti * 16 + g4 * 4 + v;
                const int64_t gr = row0 + lr;
                if (gr >= m) continue;
                const double nrm = norm_s[lr];
                const double tau = kTauRel * nrm + kTauAbs;
#pragma unroll
                for (int tj = 0; tj < 2; ++tj) {
                    const int col = col0 + wc * 32 + tj * 16 + l16;
                    if (col >= d) continue;
                    const double y = accd[ti][tj][v];
                    int code;
                    bool flag = false;
                    if (nrm == 0.0) {
                        code = L / 2;
                    } else {
                        // threshold i of this coordinate, before scaling by n
                        auto thr = [&](int i) {
                            if (!qa.athr) return bnd_s[i];
                            return athr_lds ? athr_s[i * BN + (col - col0)]
                                            : qa.athr[(int64_t)i * d + col];
                        };
                        int c = 0;
                        for (int step = L / 2; step >= 1; step >>= 1) {
                            if (c + step <= L - 1) {
                                const double t = thr(c + step - 1) * nrm;
                                if (t <= y) c += step;
                            }
                        }
                        code = c;
                        if (!std::isfinite(y)) {
                            flag = true;
                        } else {
                            if (c > 0 && y - thr(c - 1) * nrm <= tau) flag = true;
                            if (c < L - 1 && thr(c) * nrm - y <= tau) flag = true;
                        }
                    }
                    qa.codes_tmp[gr * d + col] = (uint8_t)code;
                    if (flag) {
                        // a slot of this tile's list (an LDS counter)
                        const unsigned int slot = atomicAdd(&nflag_s, 1u);
                        tflags[slot] = ((uint32_t)lr << 7) | (uint32_t)(col - col0);
                    }
                }
            }
        __syncthreads();
        if (tid == 0) qa.tile_count[tile] = nflag_s;
    } else {
#pragma unroll
        for (int ti = 0; ti < 4; ++ti)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int lr = wr * 64 + ti * 16 + g4 * 4 + v;
                const int64_t gr = row0 + lr;
                if (gr >= m) continue;
#pragma unroll
                for (int tj = 0; tj < 2; ++tj) {
                    const int col = col0 + wc * 32 + tj * 16 + l16;
                    if (col < d) fa.Y[gr * d + col] = (float)accd[ti][tj][v];
                }
            }
    }
}

// The code of coordinate j of a row with norm nrm whose exact sum is S.
__device__ inline int exact_code(double S, double nrm, int j, int d, const double *bounds,
                                 const double *athr, int levels) {
    int c = 0;
    for (int t = 0; t < levels - 1; ++t) {
        const double th = (athr ? athr[(int64_t)t * d + j] : bounds[t]) * nrm;
        c += (th <= S) ? 1 : 0;
    }
    return c;
}

// Exact recomputation of flagged coordinates, one thread per flag (one
// workgroup per output tile): the sequential float64 sum of the definition
// (products of float32 values are exact in float64, so fused and unfused
// multiply-adds agree).
__global__ __launch_bounds__(256) void fixup_kernel(
    const float *__restrict__ X, const float *__restrict__ R, int d, int ncol,
    const double *__restrict__ bounds, const double *__restrict__ athr, int levels,
    const double *__restrict__ norms,
    const uint32_t *__restrict__ flags, const unsigned int *__restrict__ tile_count,
    uint8_t *__restrict__ codes_tmp) {
    const int tile = blockIdx.x;
    const int64_t row0 = (int64_t)(tile / ncol) * BM;
    const int col0 = (tile % ncol) * BN;
    const unsigned int cnt = tile_count[tile];
    const uint32_t *tflags = flags + (int64_t)tile * (BM * BN);
    for (unsigned int e = threadIdx.x; e < cnt; e += blockDim.x) {
        const uint32_t f = tflags[e];
        const int64_t row = row0 + (f >> 7);
        const int j = col0 + (int)(f & 127);
        const f4 *xr = reinterpret_cast<const f4 *>(X + row * d);
        const f4 *rr = reinterpret_cast<const f4 *>(R + (int64_t)j * d);
        double S = 0.0;
        for (int q = 0; q < d / 4; ++q) {
            const f4 a = rr[q];
            const f4 b = xr[q];
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const double prod = (double)a[c] * (double)b[c];
                S = S + prod;
            }
        }
        codes_tmp[row * d + j] = (uint8_t)exact_code(S, norms[row], j, d, bounds, athr, levels);
    }
}

// The same recomputation for tiles with many flags: the tile's X rows and R
// rows pass through LDS in slabs of KB (once per 512 flags), and each
// thread adds its flag's products in k order from there.
__global__ __launch_bounds__(GEMM_THREADS) void fixup_tile_kernel(
    const float *__restrict__ X, int64_t m, const float *__restrict__ R, int d, int ncol,
    const double *__restrict__ bounds, const double *__restrict__ athr, int levels,
    const double *__restrict__ norms,
    const uint32_t *__restrict__ flags, const unsigned int *__restrict__ tile_count,
    uint8_t *__restrict__ codes_tmp) {
    __shared__ __attribute__((aligned(16))) float As[BM * LDS_STRIDE];
    __shared__ __attribute__((aligned(16))) float Bs[BN * LDS_STRIDE];
    const int tile = blockIdx.x;
    const int64_t row0 = (int64_t)(tile / ncol) * BM;
    const int col0 = (tile % ncol) * BN;
    const unsigned int cnt = tile_count[tile];
    if (cnt == 0) return;
    const uint32_t *tflags = flags + (int64_t)tile * (BM * BN);
    const int tid = threadIdx.x;
    for (unsigned int e0 = 0; e0 < cnt; e0 += GEMM_THREADS) {
        const unsigned int e = e0 + tid;
        const bool active = e < cnt;
        const uint32_t f = active ? tflags[e] : 0u;
        const int lr = (int)(f >> 7), lc = (int)(f & 127);
        double S = 0.0;
        for (int k0 = 0; k0 < d; k0 += KB) {
            __syncthreads();   // the previous slab has been read
#pragma unroll
            for (int r = 0; r < 2; ++r) {
                const int q = tid + r * GEMM_THREADS;
                const int row = q >> 3;
                const int kq = (q & 7) * 4;
                const int64_t gr = row0 + row;
                const f4 a = gr < m ? *reinterpret_cast<const f4 *>(X + gr * d + k0 + kq)
                                    : f4{0.f, 0.f, 0.f, 0.f};
                const f4 b = col0 + row < d
                                 ? *reinterpret_cast<const f4 *>(R + (int64_t)(col0 + row) * d + k0 + kq)
                                 : f4{0.f, 0.f, 0.f, 0.f};
                *reinterpret_cast<f4 *>(&As[row * LDS_STRIDE + kq]) = a;
                *reinterpret_cast<f4 *>(&Bs[row * LDS_STRIDE + kq]) = b;
            }
            __syncthreads();
            if (active) {
                const float *xa = &As[lr * LDS_STRIDE];
                const float *rb = &Bs[lc * LDS_STRIDE];
#pragma unroll
                for (int q = 0; q < KB; q += 4) {
                    const f4 a = *reinterpret_cast<const f4 *>(rb + q);
                    const f4 b = *reinterpret_cast<const f4 *>(xa + q);
#pragma unroll
                    for (int c = 0; c < 4; ++c) {
                        const double prod = (double)a[c] * (double)b[c];
                        S = S + prod;
                    }
                }
            }
        }
        if (active) {
            const int64_t row = row0 + lr;
            const int j = col0 + lc;
            codes_tmp[row * d + j] = (uint8_t)exact_code(S, norms[row], j, d, bounds, athr, levels);
        }
    }
}

// Packs PACK_ROWS rows per workgroup: scale, canonical bitstream, blocked layout.
constexpr int PACK_ROWS = 32;   // PACK_ROWS * d bytes of LDS (<= 64 KiB at d = 2048)

__global__ __launch_bounds__(256) void pack_kernel(
    const uint8_t *__restrict__ codes_tmp, int64_t m, int d, int bits,
    const double *__restrict__ cent_sq, const double *__restrict__ ysq,
    const double *__restrict__ norms,
    uint8_t *__restrict__ canon, float *__restrict__ scales,
    uint8_t *__restrict__ blocked, float *__restrict__ blocked_scales, int64_t base,
    int chunks) {
    extern __shared__ __attribute__((aligned(16))) uint8_t cs[];   // [PACK_ROWS][d]
    const int64_t r0 = (int64_t)blockIdx.x * PACK_ROWS;
    const int rows = (int)((m - r0) < PACK_ROWS ? (m - r0) : PACK_ROWS);
    const int tid = threadIdx.x;
    // stage codes (16 B per thread per step)
    const int vec_per_row = d / 16;
    for (int e = tid; e < rows * vec_per_row; e += blockDim.x) {
        const int r = e / vec_per_row, q = e % vec_per_row;
        reinterpret_cast<uint4 *>(cs + r * d)[q] =
            reinterpret_cast<const uint4 *>(codes_tmp + (r0 + r) * d)[q];
    }
    __syncthreads();
    // scale: one thread per row, j in order
    if (tid < rows) {
        const uint8_t *c = cs + tid * d;
        // sum_j fl64(yhat_j^2): c[code]^2, or with TQ+ the calibrated
        // reconstruction's square, per coordinate ([d][levels])
        const int L = 1 << bits;
        double h2 = 0.0;
        if (ysq)
            for (int j = 0; j < d; ++j) h2 = h2 + ysq[(int64_t)j * L + c[j]];
        else
            for (int j = 0; j < d; ++j) h2 = h2 + cent_sq[c[j]];
        const double nrm = norms[r0 + tid];
        const float s = (nrm == 0.0) ? 0.0f : (float)(nrm / std::sqrt(h2));
        if (scales) scales[r0 + tid] = s;
        if (blocked_scales) blocked_scales[base + r0 + tid] = s;
    }
    // canonical rows: 32-bit words, bits LSB-first
    const int wpr = d * bits / 32;   // words per canonical row
    if (canon) {
        for (int e = tid; e < rows * wpr; e += blockDim.x) {
            const int r = e / wpr, w = e % wpr;
            const uint8_t *c = cs + r * d;
            uint32_t word = 0;
            if (bits == 3) {
                const int b0 = w * 32;
                for (int t = 0; t < 32; ++t) {
                    const int bit = b0 + t;
                    const int j = bit / 3, sh = bit % 3;
                    word |= (uint32_t)((c[j] >> sh) & 1) << t;
                }
            } else {
                const int per = 32 / bits;
                for (int t = 0; t < per; ++t) word |= (uint32_t)c[w * per + t] << (t * bits);
            }
            reinterpret_cast<uint32_t *>(canon + (r0 + r) * (int64_t)(d * bits / 8))[w] = word;
        }
    }
    // blocked layout: 16-byte chunk ch of vector v at ((v/64)*chunks + ch)*1024 + (v%64)*16
    if (blocked) {
        for (int e = tid; e < rows * chunks * 4; e += blockDim.x) {
            const int r = e / (chunks * 4), rem = e % (chunks * 4);
            const int ch = rem >> 2, wq = rem & 3;
            const uint8_t *c = cs + r * d;
            uint32_t word = 0;
            if (bits == 3) {
                const int j0 = (ch * 4 + wq) * 10;
                for (int t = 0; t < 10; ++t) {
                    const int j = j0 + t;
                    if (j < d) word |= (uint32_t)c[j] << (3 * t);
                }
            } else {
                const int per = 32 / bits;
                const int j0 = (ch * 4 + wq) * per;
                for (int t = 0; t < per; ++t) word |= (uint32_t)c[j0 + t] << (t * bits);
                if (blocked_rotated(bits)) word = rotl2(word);
            }
            const int64_t v = base + r0 + r;
            uint8_t *dst = blocked + ((v >> 6) * chunks + ch) * 1024 + (v & 63) * 16;
            reinterpret_cast<uint32_t *>(dst)[wq] = word;
        }
    }
}

// Y = X R^T for a few rows (m <= kSmallRows), with exactly the arithmetic of
// rot_gemm<false>: every output element goes through the same
// v_mfma_f32_16x16x4f32 sequence (the same k in the same operand slots, sub
// and step order), its float32 partial is folded into float64 after each
// 32-wide slab and rounded to float32 at the end, so a row rotates to the
// same bits in either kernel.  One wave per 16 x 16 output block reads its
// fragments straight from memory, P slabs ahead: many small workgroups
// instead of a few 128 x 128 tiles, for the latency of short batches.
constexpr int kSmallRows = 64;

template <int P>
__global__ __launch_bounds__(256) void rot_small_kernel(const float *__restrict__ X, int64_t m,
                                                        int d, const float *__restrict__ R,
                                                        float *__restrict__ Y) {
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int l16 = lane & 15;
    const int g4 = lane >> 4;
    const int64_t r0 = (int64_t)blockIdx.y * 16;
    const int c0 = (blockIdx.x * 4 + wave) * 16;
    if (c0 >= d) return;   // no barrier in this kernel
    const int64_t gr = r0 + l16;   // the row of X this lane loads
    const bool rowok = gr < m;
    const float *xa = X + (rowok ? gr : 0) * d + g4 * 4;
    const float *rb = R + (int64_t)(c0 + l16) * d + g4 * 4;
    const int nslab = d / KB;      // even; a multiple of P
    f4 fa[P][2], fb[P][2];
    auto load = [&](int s, f4 (&A)[2], f4 (&B)[2]) {
#pragma unroll
        for (int sub = 0; sub < 2; ++sub) {
            A[sub] = rowok ? *reinterpret_cast<const f4 *>(xa + s * KB + sub * 16)
                           : f4{0.f, 0.f, 0.f, 0.f};
            B[sub] = *reinterpret_cast<const f4 *>(rb + s * KB + sub * 16);
        }
    };
#pragma unroll
    for (int u = 0; u < P; ++u) load(u, fa[u], fb[u]);
    f4 acc = f4{0.f, 0.f, 0.f, 0.f};
    double accd[4] = {0.0, 0.0, 0.0, 0.0};
    for (int s0 = 0; s0 < nslab; s0 += P) {
#pragma unroll
        for (int u = 0; u < P; ++u) {
#pragma unroll
            for (int sub = 0; sub < 2; ++sub)
#pragma unroll
                for (int st = 0; st < 4; ++st)
                    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[u][sub][st], fb[u][sub][st],
                                                               acc, 0, 0, 0);
#pragma unroll
            for (int v = 0; v < 4; ++v) accd[v] += (double)acc[v];
            acc = f4{0.f, 0.f, 0.f, 0.f};
            if (s0 + u + P < nslab) load(s0 + u + P, fa[u], fb[u]);
        }
    }
#pragma unroll
    for (int v = 0; v < 4; ++v) {
        const int64_t row = r0 + g4 * 4 + v;
        if (row < m) Y[row * d + c0 + l16] = (float)accd[v];
    }
}

}  // namespace

// Output tiles of one chunk of rows.
size_t encode_tiles(int d) {
    return (size_t)(kEncodeChunkRows / BM) * (size_t)((d + BN - 1) / BN);
}

size_t encode_workspace_bytes(int d) {
    const size_t rows = kEncodeChunkRows;
    size_t b = 0;
    b += rows * (size_t)d;                    // unpacked codes
    b = (b + 255) & ~(size_t)255;
    b += rows * sizeof(double);               // norms
    b = (b + 255) & ~(size_t)255;
    b += encode_tiles(d) * BM * BN * sizeof(uint32_t);   // flags (worst case: every coordinate)
    b = (b + 255) & ~(size_t)255;
    b += encode_tiles(d) * sizeof(unsigned int);          // flags per tile
    b = (b + 255) & ~(size_t)255;
    b += 255 * sizeof(double) + 256 * sizeof(double);   // bounds, cent_sq
    b = (b + 255) & ~(size_t)255;
    return b;
}

hipError_t encode_rows(const float *X, int64_t n, int d, const float *R,
                       const CodebookDev &cb, const EncodeOut &out, void *ws,
                       int *status_dev, hipStream_t stream, const CalibDev &calib) {
    const size_t rows = kEncodeChunkRows;
    uint8_t *p = static_cast<uint8_t *>(ws);
    uint8_t *codes_tmp = p;
    p += (rows * (size_t)d + 255) & ~(size_t)255;
    double *norms = reinterpret_cast<double *>(p);
    p += (rows * sizeof(double) + 255) & ~(size_t)255;
    uint32_t *flags = reinterpret_cast<uint32_t *>(p);
    p += (encode_tiles(d) * BM * BN * sizeof(uint32_t) + 255) & ~(size_t)255;
    unsigned int *tile_count = reinterpret_cast<unsigned int *>(p);
    p += (encode_tiles(d) * sizeof(unsigned int) + 255) & ~(size_t)255;
    double *bounds = reinterpret_cast<double *>(p);
    double *cent_sq = bounds + 255;

    hipError_t e = hipMemcpyAsync(bounds, cb.bounds, sizeof(double) * (cb.levels - 1),
                                  hipMemcpyHostToDevice, stream);
    if (e != hipSuccess) return e;
    e = hipMemcpyAsync(cent_sq, cb.cent_sq, sizeof(double) * cb.levels,
                       hipMemcpyHostToDevice, stream);
    if (e != hipSuccess) return e;

    const int chunks = chunks_per_vector(d, cb.bits);
    const int ncol = (d + BN - 1) / BN;
    for (int64_t r0 = 0; r0 < n; r0 += rows) {
        const int64_t m = (n - r0) < (int64_t)rows ? (n - r0) : (int64_t)rows;
        const int nrt = (int)((m + BM - 1) / BM);
        const int groups = (nrt + 7) / 8;
        // every output tile of the chunk writes its flag count
        QuantArgs qa{bounds, calib.athr, cb.levels, codes_tmp, norms, flags, tile_count, status_dev};
        F32Args fa{nullptr};
        hipLaunchKernelGGL((rot_gemm<true>), dim3(groups * 8 * ncol), dim3(GEMM_THREADS), 0,
                           stream, X + r0 * d, m, R, d, nrt, qa, fa);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        // 8-bit codes flag about 2% of coordinates (thresholds ~4e-4 apart
        // at d = 1536): tiles then share their staged rows
        if (cb.levels > 16)
            hipLaunchKernelGGL(fixup_tile_kernel, dim3(nrt * ncol), dim3(GEMM_THREADS), 0, stream,
                               X + r0 * d, m, R, d, ncol, bounds, calib.athr, cb.levels, norms,
                               flags, tile_count, codes_tmp);
        else
            hipLaunchKernelGGL(fixup_kernel, dim3(nrt * ncol), dim3(256), 0, stream, X + r0 * d, R,
                               d, ncol, bounds, calib.athr, cb.levels, norms, flags, tile_count,
                               codes_tmp);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        const int packs = (int)((m + PACK_ROWS - 1) / PACK_ROWS);
        hipLaunchKernelGGL(pack_kernel, dim3(packs), dim3(256), PACK_ROWS * d, stream,
                           codes_tmp, m, d, cb.bits, cent_sq, calib.ysq, norms,
                           out.canonical ? out.canonical + r0 * (int64_t)(d * cb.bits / 8) : nullptr,
                           out.scales ? out.scales + r0 : nullptr, out.blocked,
                           out.blocked_scales, out.base + r0, chunks);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t rotate_rows_f32(const float *X, int64_t m, int d, const float *R, float *Y,
                           hipStream_t stream) {
    if (m <= 0) return hipSuccess;
    if (m <= kSmallRows) {
        const dim3 grid((unsigned)((d + 63) / 64), (unsigned)((m + 15) / 16));
        if ((d / KB) % 4 == 0)
            hipLaunchKernelGGL(rot_small_kernel<4>, grid, dim3(256), 0, stream, X, m, d, R, Y);
        else
            hipLaunchKernelGGL(rot_small_kernel<2>, grid, dim3(256), 0, stream, X, m, d, R, Y);
        return hipGetLastError();
    }
    const int ncol = (d + BN - 1) / BN;
    const int nrt = (int)((m + BM - 1) / BM);
    const int groups = (nrt + 7) / 8;
    QuantArgs qa{};
    F32Args fa{Y};
    hipLaunchKernelGGL((rot_gemm<false>), dim3(groups * 8 * ncol), dim3(GEMM_THREADS), 0,
                       stream, X, m, R, d, nrt, qa, fa);
    return hipGetLastError();
}

}  // namespace tq
