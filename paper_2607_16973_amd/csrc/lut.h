// Per-query lookup tables for 4-bit fields of the code stream (b in
// {1, 2, 4}) and for 3-bit codes (b = 3), and the integer scoring that uses
// them (device code, shared by the single-query scan and the exact
// rescoring of the batched search).
//
// One row of 16 int32 entries per 4-bit field of the code stream (row r
// covers coordinates r*g .. r*g+g-1, g = 4/b), holding round(2^sh * sum_t
// c[code_t] q'_j) -- fixed point with a per-query power of two 2^sh chosen so
// that every possible sum of one entry per row fits in int32: sum_r max_c
// |entry| <= 2^sh max|c| sum_j |q'_j| + rows/2 < 2^31.  The integer sums are
// then exact and independent of summation order.  A vector's score is
// s * (float)sum * 2^-sh, computed the same way wherever it is needed.
// With TQ+ calibration (section II-B) the reconstruction is mu_j + kappa_j c,
// so the table is built from q''_j = kappa_j q'_j and every entry of row 0
// also holds round(2^sh C), C = sum_j mu_j q'_j: each code hits row 0 once,
// so every sum carries C exactly once.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace tq {

// Threads of a workgroup that builds a table, and its waves.
constexpr int kTableThreads = 1024;
constexpr int kTableWaves = kTableThreads / 64;

struct TableShape {
    int d, bits;
    int lut_words;   // 32-bit words of the table: d * b * 4
};

// Sum of 8 int32 table hits addressed by the 8 4-bit fields of a stored
// word w (the canonical word rotated left by 2 bits); row t of the 8 rows
// starting at Lb (64 bytes per row) is indexed by field t.
__device__ inline int nib8(const char *__restrict__ Lb, uint32_t w) {
    uint32_t lo = w & 0x3C3C3C3Cu;                                  // byte b: field 2b   times 4
    uint32_t hi = __builtin_amdgcn_alignbit(w, w, 4) & 0x3C3C3C3Cu; // byte b: field 2b+1 times 4
    // keep the byte-aligned form: each address is then one add with a byte
    // select (SDWA) instead of a shift, a mask and an add per field
    asm volatile("" : "+v"(lo), "+v"(hi));
    const int a0 = *reinterpret_cast<const int *>(Lb + 0 * 64 + (lo & 0xFFu));
    const int a1 = *reinterpret_cast<const int *>(Lb + 1 * 64 + (hi & 0xFFu));
    const int a2 = *reinterpret_cast<const int *>(Lb + 2 * 64 + ((lo >> 8) & 0xFFu));
    const int a3 = *reinterpret_cast<const int *>(Lb + 3 * 64 + ((hi >> 8) & 0xFFu));
    const int a4 = *reinterpret_cast<const int *>(Lb + 4 * 64 + ((lo >> 16) & 0xFFu));
    const int a5 = *reinterpret_cast<const int *>(Lb + 5 * 64 + ((hi >> 16) & 0xFFu));
    const int a6 = *reinterpret_cast<const int *>(Lb + 6 * 64 + (lo >> 24));
    const int a7 = *reinterpret_cast<const int *>(Lb + 7 * 64 + (hi >> 24));
    return (a0 + a1 + a2) + (a3 + a4 + a5) + (a6 + a7);
}

// Sum of the 32 table hits of one 16-byte chunk; Lb is the chunk's 2 KiB of
// table rows.
__device__ inline int nib_chunk(const char *__restrict__ Lb, uint4 v) {
    return (nib8(Lb, v.x) + nib8(Lb + 512, v.y)) + (nib8(Lb + 1024, v.z) + nib8(Lb + 1536, v.w));
}

__device__ inline float wave_sum(float v) {
#pragma unroll
    for (int m = 32; m > 0; m >>= 1) v += __shfl_xor(v, m, 64);
    return v;
}

// 4-bit-field tables (b in {1, 2, 4}): row r of 16 entries covers
// coordinates r*g .. r*g+g-1 (g = 4/b) and rows = d*b/4 <= 2048, so thread t
// owns rows t and t + 1024.  Loads the thread's coordinates of q'.
__device__ inline void load_nibble_query(const TableShape &p, const float *__restrict__ q,
                                         float (&qv)[2][4]) {
    const int g = 4 / p.bits;
    const int rows = p.lut_words >> 4;
#pragma unroll
    for (int m = 0; m < 2; ++m) {
        const int r = threadIdx.x + m * kTableThreads;
#pragma unroll
        for (int t = 0; t < 4; ++t) qv[m][t] = (r < rows && t < g) ? q[r * g + t] : 0.f;
    }
}

// Writes this wave's share of sum_j |q'_j| to red[wave] (16 floats of LDS).
__device__ inline void nibble_abs_sum(float *red, const float (&qv)[2][4]) {
    float part = 0.f;
#pragma unroll
    for (int m = 0; m < 2; ++m)
#pragma unroll
        for (int t = 0; t < 4; ++t) part += fabsf(qv[m][t]);
    part = wave_sum(part);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = part;
}

// Writes the int32 table from the coordinates loaded by load_nibble_query,
// once red[] holds the 16 wave sums of |q'| (nibble_abs_sum, then a
// barrier); returns the table's exponent sh.  The caller synchronises
// before the table is read.
//
// Entries are rounded from float32 products: each is within 1/2 unit of
// 2^sh c q' plus 2^-23 of its magnitude, so the summed error stays below
// 2^-23 B + rows/2 + 1 units, B = max|c| sum_j |q'_j| + |C| -- far inside the
// score tolerance.  C is the query's constant term (0 without calibration).
__device__ inline int build_nibble_table(float *lds, const float *red, const float *cents,
                                         const TableShape &p, const float (&qv)[2][4],
                                         float C = 0.f) {
    const int tid = threadIdx.x;
    const int rows = p.lut_words >> 4;
    const int L = 1 << p.bits;
    // the levels: at most 16 (`cents` holds 16 values, unused ones finite)
    float cl[16];
#pragma unroll
    for (int c = 0; c < 16; ++c) cl[c] = cents[c];
    double tot = 0.0;
#pragma unroll
    for (int w = 0; w < kTableWaves; ++w) tot += (double)red[w];
    const double cmax = fmax(fabs((double)cl[0]), fabs((double)cl[L - 1]));
    // bound with margin for the float32 partial sums and products
    const double B = (cmax * tot + fabs((double)C)) * (1.0 + 1e-5);
    int sh = 0;
    if (B > 0.0) {
        sh = (int)floor(log2((2147483647.0 - 2.0 * p.d) / B));
        sh = sh < 0 ? 0 : (sh > 100 ? 100 : sh);
    }
    const float scale = ldexpf(1.0f, sh);
    const int c0 = (int)rintf(C * scale);
    int *T = reinterpret_cast<int *>(lds);
#pragma unroll
    for (int m = 0; m < 2; ++m) {
        const int r = tid + m * kTableThreads;
        if (r < rows) {
            const float q0 = qv[m][0] * scale, q1 = qv[m][1] * scale;
            const float q2 = qv[m][2] * scale, q3 = qv[m][3] * scale;
            int e[16];
            if (p.bits == 4) {
#pragma unroll
                for (int c = 0; c < 16; ++c) e[c] = (int)rintf(cl[c] * q0);
            } else if (p.bits == 2) {
#pragma unroll
                for (int c = 0; c < 16; ++c) e[c] = (int)rintf(fmaf(cl[c & 3], q0, cl[c >> 2] * q1));
            } else {
#pragma unroll
                for (int c = 0; c < 16; ++c)
                    e[c] = (int)rintf(fmaf(cl[c & 1], q0, cl[(c >> 1) & 1] * q1) +
                                      fmaf(cl[(c >> 2) & 1], q2, cl[c >> 3] * q3));
            }
            if (r == 0)
#pragma unroll
                for (int c = 0; c < 16; ++c) e[c] += c0;
            int4 *row = reinterpret_cast<int4 *>(T + r * 16);
#pragma unroll
            for (int c4 = 0; c4 < 4; ++c4)
                row[c4] = make_int4(e[4 * c4], e[4 * c4 + 1], e[4 * c4 + 2], e[4 * c4 + 3]);
        }
    }
    return sh;
}

// ---------------------------------------------------------------- b = 3
// Stored words hold ten 3-bit fields (bits 3t..3t+2: coordinate 10w + t of
// the word's run; two pad bits), so a 16-byte chunk covers 40 coordinates.
// The table has one row of 8 int32 entries (32 bytes) per coordinate,
// round(2^sh c[code] q'_j), under the same fixed-point rule as the 4-bit
// field tables; rows = chunks * 40 <= 3 * 1024 (d <= 2048), so thread t owns
// rows t, t + 1024 and t + 2048, and rows of padding coordinates (j >= d)
// are zero.  With TQ+ calibration row 0 also carries round(2^sh C).
constexpr int kTriRowsPerThread = 3;

__device__ inline void load_tribit_query(const TableShape &p, const float *__restrict__ q,
                                         float (&qv)[kTriRowsPerThread]) {
#pragma unroll
    for (int m = 0; m < kTriRowsPerThread; ++m) {
        const int j = threadIdx.x + m * kTableThreads;
        qv[m] = j < p.d ? q[j] : 0.f;
    }
}

__device__ inline void tribit_abs_sum(float *red, const float (&qv)[kTriRowsPerThread]) {
    float part = 0.f;
#pragma unroll
    for (int m = 0; m < kTriRowsPerThread; ++m) part += fabsf(qv[m]);
    part = wave_sum(part);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = part;
}

// As build_nibble_table, for the 3-bit rows; the summed rounding error
// stays below 2^-23 B + d/2 + 1 units.
__device__ inline int build_tribit_table(float *lds, const float *red, const float *cents,
                                         const TableShape &p, const float (&qv)[kTriRowsPerThread],
                                         float C = 0.f) {
    const int tid = threadIdx.x;
    const int rows = p.lut_words >> 3;
    float cl[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) cl[c] = cents[c];
    double tot = 0.0;
#pragma unroll
    for (int w = 0; w < kTableWaves; ++w) tot += (double)red[w];
    const double cmax = fmax(fabs((double)cl[0]), fabs((double)cl[7]));
    const double B = (cmax * tot + fabs((double)C)) * (1.0 + 1e-5);
    int sh = 0;
    if (B > 0.0) {
        sh = (int)floor(log2((2147483647.0 - 2.0 * p.d) / B));
        sh = sh < 0 ? 0 : (sh > 100 ? 100 : sh);
    }
    const float scale = ldexpf(1.0f, sh);
    const int c0 = (int)rintf(C * scale);
    int *T = reinterpret_cast<int *>(lds);
#pragma unroll
    for (int m = 0; m < kTriRowsPerThread; ++m) {
        const int r = tid + m * kTableThreads;
        if (r < rows) {
            const float q0 = qv[m] * scale;
            int e[8];
#pragma unroll
            for (int c = 0; c < 8; ++c) e[c] = (int)rintf(cl[c] * q0);
            if (r == 0)
#pragma unroll
                for (int c = 0; c < 8; ++c) e[c] += c0;
            int4 *row = reinterpret_cast<int4 *>(T + r * 8);
            row[0] = make_int4(e[0], e[1], e[2], e[3]);
            row[1] = make_int4(e[4], e[5], e[6], e[7]);
        }
    }
    return sh;
}

// Sum of the 10 table hits of one stored word; Lb is its 10 rows (320 bytes).
// Each address is a bit-field extract and a shift-add onto Lb (the empty asm
// keeps the compiler from re-forming them into a shift, a mask and an add).
__device__ inline int tri10(const char *__restrict__ Lb, uint32_t w) {
    int a = 0, b = 0;
#pragma unroll
    for (int t = 0; t < 10; t += 2) {
        uint32_t f0 = __builtin_amdgcn_ubfe(w, 3 * t, 3);
        uint32_t f1 = __builtin_amdgcn_ubfe(w, 3 * t + 3, 3);
        asm volatile("" : "+v"(f0), "+v"(f1));
        a += *reinterpret_cast<const int *>(Lb + t * 32 + (f0 << 2));
        b += *reinterpret_cast<const int *>(Lb + (t + 1) * 32 + (f1 << 2));
    }
    return a + b;
}

// Sum of the 40 table hits of one 16-byte chunk; Lb is the chunk's 1280
// bytes of table rows.
__device__ inline int tri_chunk(const char *__restrict__ Lb, uint4 v) {
    return (tri10(Lb, v.x) + tri10(Lb + 320, v.y)) + (tri10(Lb + 640, v.z) + tri10(Lb + 960, v.w));
}

}  // namespace tq
