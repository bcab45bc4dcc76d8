// Rotation + quantisation of float32 rows on gfx950 (section II-B, steps 1-5).
//
// Pipeline per chunk of rows:
//  0. row_norm_kernel: the exact row norm n = sqrt(sum_k x_k^2) (sequential
//     float64 over k) and a report of non-finite inputs.
//  1. encode_gemm: Y = X R^T on the matrix cores (v_mfma_f32_32x32x2f32),
//     with each 32-wide slab of k accumulated in float32 and then added into
//     float64 accumulators.  The epilogue turns every y into a code by
//     comparing it with fl64(t_i * n) and flags the coordinate when y lies
//     within tau of a threshold, where tau bounds |y - S| for S the float64
//     sequential dot product of the definition:
//       per slab, float32 MFMA accumulation of 32 products from 0, in any
//       order:
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
#include <type_traits>

#include "kernels.h"
#include "lds_dma.h"

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

// XCD-aware tile order: the d/BN column tiles of one row tile go to the same
// XCD (workgroups are dealt to the 8 XCDs round-robin), so the X tile is read
// from HBM once and then served by that XCD's L2.
__device__ inline void tile_of(int bid, int ncol, int &rt, int &ct) {
    const int x = bid & 7;
    const int rest = bid >> 3;
    ct = rest % ncol;
    rt = (rest / ncol) * 8 + x;
}

// Y = X R^T in float32 (query rotation).  Each 32-wide k-slab is
// accumulated on the matrix cores (v_mfma_f32_16x16x4f32, lane (l16, g4)
// feeding k = 16 sub + 4 g4 + st to step st of sub-slab sub) and then added
// into float64 accumulators in slab order; the result is rounded to float32
// once.  rot_small_kernel repeats exactly this arithmetic.
__global__ __launch_bounds__(GEMM_THREADS) void rot_gemm(
    const float *__restrict__ X, int64_t m, const float *__restrict__ R, int d,
    int n_row_tiles, float *__restrict__ Y) {
    __shared__ __attribute__((aligned(16))) float As[2][BM * LDS_STRIDE];
    __shared__ __attribute__((aligned(16))) float Bs[2][BN * LDS_STRIDE];

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

    const int nslab = d / KB;
    load_slab(0);
    store_slab(0);
    __syncthreads();
    for (int s = 0; s < nslab; ++s) {
        const int buf = s & 1;
        if (s + 1 < nslab) load_slab((s + 1) * KB);
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
                if (col < d) Y[gr * d + col] = (float)accd[ti][tj][v];
            }
        }
}

// ------------------------------------------------------------- row norms
// n = sqrt(sum_k x_k^2) of every row of the chunk: one thread per row adds
// the squares in k order in float64 (x^2 is exact in float64, so the fused
// multiply-add rounds exactly as add(fl(x^2))).  A wave takes 64 rows in
// slabs of RN_KS coordinates: every load instruction reads the 256-byte
// slabs of 4 rows, the slab passes through LDS (rows padded to 17 pieces, so
// the summing lanes read distinct banks), and lane r adds row r's squares;
// two slabs are in registers while one is summed.  A non-finite input makes
// the sum non-finite (x^2 of a finite float32 cannot overflow float64),
// which sets *status.
constexpr int RN_KS = 64;               // coordinates per slab (d is a multiple of 64)
constexpr int RN_PQ = RN_KS / 4;        // 16-byte pieces of a row slab
constexpr int RN_LD = 64 * RN_PQ / 64;  // load instructions per slab (4 rows each)

struct RnSlab {
    f4 v[RN_LD];
};

__global__ __launch_bounds__(64) void row_norm_kernel(const float *__restrict__ X, int64_t m,
                                                      int d, double *__restrict__ norms,
                                                      int *__restrict__ status) {
    constexpr int PS = RN_PQ + 1;
    __shared__ f4 xs[64 * PS];
    const int lane = threadIdx.x;
    const int64_t r0 = (int64_t)blockIdx.x * 64;
    const int ns = d / RN_KS;
    // load i: lanes 16 g .. 16 g + 15 read row 4 i + g (rows past m: the last)
    auto row_ptr = [&](int i) {
        int64_t r = r0 + 4 * i + (lane >> 4);
        r = r < m ? r : m - 1;
        return X + r * d + 4 * (lane & 15);
    };
    auto load = [&](int sl, RnSlab &b) {
#pragma unroll
        for (int i = 0; i < RN_LD; ++i)
            b.v[i] = *reinterpret_cast<const f4 *>(row_ptr(i) + sl * RN_KS);
    };
    // the barriers order the lanes' LDS accesses (a lane sums what other
    // lanes staged) and leave the loads in flight
    auto stage = [&](const RnSlab &b) {
        lds_barrier();
#pragma unroll
        for (int i = 0; i < RN_LD; ++i) xs[(4 * i + (lane >> 4)) * PS + (lane & 15)] = b.v[i];
        lds_barrier();
        // the refill of these registers stays after the writes: moved ahead,
        // it would take other registers and the loop would copy them back
        // at its back edge, waiting for every load in flight
        __builtin_amdgcn_sched_barrier(0);
    };
    double s2 = 0.0;
    auto sum = [&]() {
#pragma unroll
        for (int q = 0; q < RN_PQ; ++q) {
            const f4 v = xs[lane * PS + q];
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const double x = (double)v[c];
                s2 = __builtin_fma(x, x, s2);
            }
        }
    };
    RnSlab b0, b1;
    load(0, b0);
    __builtin_amdgcn_sched_barrier(0);   // b0's loads all ahead of b1's
    load(ns > 1 ? 1 : 0, b1);
    for (int sl = 0; sl < ns; sl += 2) {
        stage(b0);
        load(sl + 2 < ns ? sl + 2 : ns - 1, b0);
        sum();
        if (sl + 1 < ns) stage(b1);
        load(sl + 3 < ns ? sl + 3 : ns - 1, b1);
        if (sl + 1 < ns) sum();
    }
    const int64_t r = r0 + lane;
    if (r < m) {
        norms[r] = std::sqrt(s2);
        if (!std::isfinite(s2)) atomicOr(status, 1);
    }
}

// ------------------------------------------------------------- encode_gemm
// Y = X R^T with the quantiser epilogue, for the encode.  Same tiles and
// workgroup shape as rot_gemm (128 x 128, k-slabs of 32, 8 waves of 64 x 32),
// but built for throughput:
//  - v_mfma_f32_32x32x2f32 (two 32 x 32 tiles per wave), which keeps the
//    matrix pipe busier than 16x16x4 at two waves per SIMD;
//  - a four-stage LDS ring filled by direct global -> LDS loads three slabs
//    ahead, one barrier per slab, and each k-group's operands read from LDS
//    one group ahead, so that no load or LDS latency sits between a barrier
//    and the next MFMA;
//  - two sets of float32 accumulators: the float64 fold of slab s-1 is
//    interleaved with the MFMAs of slab s;
//  - the row norms come from row_norm_kernel (float64 vector work in this
//    loop does not overlap the matrix pipe).
// Slab s covers k in [32s, 32s+32); group g of it k in [32s+8g, 32s+8g+8).
// Lane l (h = l / 32) of a wave feeds k = 32s + 8g + 4h + t to step t of
// group g, so one 16-byte LDS read per operand and group serves 4 MFMAs.
// The float32 partial of a slab sums its 32 products in an order of the
// matrix core's choosing; the error bound behind tau (any order of a
// 32-term float32 sum from zero) is the same as for rot_gemm.
constexpr int EG_STAGES = 4;
constexpr int EG_OPER_B = BM * KB * 4;   // bytes of one operand tile of a slab (16 KiB)
constexpr int EG_STAGE_B = 2 * EG_OPER_B;  // A then B

// Operand tiles are stored unpadded in four planes, one per k-group g:
// plane g holds, for each of the 128 rows, the row's floats 8g .. 8g+7 of
// the slab as two 16-byte pieces, piece h at byte 4096 g + 32 r +
// 16 (h ^ eg_swz(r)).  A read of piece h of 16 consecutive rows (8, with
// 32 banks) then meets distinct banks, and the group index is an immediate
// offset.
__device__ inline int eg_swz(int r) { return ((r >> 2) ^ (r >> 3)) & 1; }

typedef float f16v __attribute__((ext_vector_type(16)));

__global__ __launch_bounds__(GEMM_THREADS) void encode_gemm(
    const float *__restrict__ X, int64_t m, const float *__restrict__ R, int d,
    int n_row_tiles, QuantArgs qa) {
    __shared__ __attribute__((aligned(1024))) char stg[EG_STAGES * EG_STAGE_B];
    __shared__ double norm_s[BM];
    __shared__ double bnd_s[255];
    __shared__ double athr_s[15 * BN];   // TQ+ thresholds of the tile's columns, b <= 4
    __shared__ unsigned int nflag_s;

    const int ncol = (d + BN - 1) / BN;
    int rt, ct;
    tile_of(blockIdx.x, ncol, rt, ct);
    if (rt >= n_row_tiles) return;
    const int64_t row0 = (int64_t)rt * BM;
    const int col0 = ct * BN;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wr = wave >> 2;     // 0..1 : 64-row half
    const int wc = wave & 3;      // 0..3 : 32-column quarter
    const int l32 = lane & 31;
    const int h = lane >> 5;
    const int nslab = d / KB;     // even: d is a multiple of 64

    // This wave's loads of a slab: pieces 128 wave + 64 j + lane (j = 0, 1)
    // of the A tile and of the B tile.  Rows of X past m and rows of R past
    // d are clamped to the last one: they only feed outputs the epilogue
    // drops.
    // This wave's loads of a slab: 1 KiB pieces 2 wave + j (j = 0, 1) of the
    // A tile and of the B tile, i.e. plane wave / 2, rows 32 ((2 wave + j) & 3)
    // + lane / 2.  Rows of X past m and rows of R past d are clamped to the
    // last one: they only feed outputs that the epilogue drops.
    uint32_t off_a[2], off_b[2];   // byte offsets of the lane's pieces in slab 0
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int i = 2 * wave + j;
        const int row = 32 * (i & 3) + (lane >> 1);
        const int k = 8 * (i >> 2) + 4 * ((lane & 1) ^ eg_swz(row));
        const int64_t ar = row0 + row < m ? row0 + row : m - 1;
        const int br = col0 + row < d ? col0 + row : d - 1;
        off_a[j] = (uint32_t)((ar * d + k) * 4);
        off_b[j] = (uint32_t)(((int64_t)br * d + k) * 4);
    }
    const uint32_t stg_lds = (uint32_t)(uintptr_t)stg;
    // slab s into stage ST: 4 loads per wave (uniform base + 32-bit lane offset)
    auto request = [&](int s, auto ST) {
        constexpr uint32_t stage = decltype(ST)::value;
        const uint32_t base = stg_lds + stage * EG_STAGE_B + (uint32_t)wave * 2048;
        const float *xa = X + s * KB;
        const float *rb = R + s * KB;
        lds_dma16_s(off_a[0], xa, base);
        lds_dma16_s(off_a[1], xa, base + 1024);
        lds_dma16_s(off_b[0], rb, base + EG_OPER_B);
        lds_dma16_s(off_b[1], rb, base + EG_OPER_B + 1024);
    };
    // operands of group g: A rows of the wave's two 32-row tiles, B columns
    const int pz = 16 * (h ^ eg_swz(l32));   // eg_swz(row) of every row this lane reads
    const int a_base = (wr * 64 + l32) * 32 + pz;
    const int b_base = EG_OPER_B + (wc * 32 + l32) * 32 + pz;
    auto opread = [&](auto ST, int g, f4 &a0, f4 &a1, f4 &b) {
        constexpr int stage = decltype(ST)::value;
        const char *S = stg + stage * EG_STAGE_B + 4096 * g;
        a0 = *reinterpret_cast<const f4 *>(S + a_base);
        a1 = *reinterpret_cast<const f4 *>(S + a_base + 32 * 32);
        b = *reinterpret_cast<const f4 *>(S + b_base);
    };

    if (!qa.athr)
        for (int i = tid; i < qa.levels - 1; i += GEMM_THREADS) bnd_s[i] = qa.bounds[i];
    const bool athr_lds = qa.athr && qa.levels <= 16;
    if (athr_lds)
        for (int e = tid; e < (qa.levels - 1) * BN; e += GEMM_THREADS) {
            const int i = e / BN, c = col0 + e % BN;
            athr_s[e] = c < d ? qa.athr[(int64_t)i * d + c] : 0.0;
        }
    if (tid == 0) nflag_s = 0;
    if (tid < BM) norm_s[tid] = row0 + tid < m ? qa.norms[row0 + tid] : 0.0;

    // prologue: slabs 0, 1 and 2 requested, 0 and 1 landed
    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;
    using I2 = std::integral_constant<int, 2>;
    using I3 = std::integral_constant<int, 3>;
    request(0, I0());
    request(1, I1());
    if (nslab > 2) {
        request(2, I2());
        wait_vmem<4>();
    } else {
        wait_vmem<0>();
    }
    lds_barrier();

    const f16v zero = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f,
                       0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    f16v acc[2][2];     // [set][tile]: float32 partials of slab s (set s & 1)
    double accd[2][16]; // [tile][i]
#pragma unroll
    for (int t = 0; t < 2; ++t) {
        acc[1][t] = zero;
#pragma unroll
        for (int i = 0; i < 16; ++i) accd[t][i] = 0.0;
    }
    // operands: set g & 1 feeds group g while group g + 1's are read into
    // the other set (static indices once unrolled: no register copies)
    f4 op[2][3];
    opread(I0(), 0, op[0][0], op[0][1], op[0][2]);

    // slab s, held in stage ST (static, so that every LDS address is an
    // offset from a fixed register)
    auto slab = [&](int s, auto ST, f16v(&cur)[2], const f16v(&prv)[2]) {
        using Next = std::integral_constant<int, (decltype(ST)::value + 1) % EG_STAGES>;
        using Far = std::integral_constant<int, (decltype(ST)::value + 3) % EG_STAGES>;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            f4(&c)[3] = op[g & 1];
            f4(&n)[3] = op[(g + 1) & 1];
            if (g < 3)
                opread(ST, g + 1, n[0], n[1], n[2]);
            else if (s + 1 < nslab)
                opread(Next(), 0, n[0], n[1], n[2]);
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                cur[0] = __builtin_amdgcn_mfma_f32_32x32x2f32(c[0][t], c[2][t],
                                                              (g == 0 && t == 0) ? zero : cur[0], 0, 0, 0);
                cur[1] = __builtin_amdgcn_mfma_f32_32x32x2f32(c[1][t], c[2][t],
                                                              (g == 0 && t == 0) ? zero : cur[1], 0, 0, 0);
            }
            // fold a quarter of slab s-1's partials (zeros before slab 0)
#pragma unroll
            for (int i = 0; i < 8; ++i)
                accd[g >> 1][(g & 1) * 8 + i] += (double)prv[g >> 1][(g & 1) * 8 + i];
            if (g == 1) {
                // slab s+1 has landed (this wave's loads; the barrier makes it
                // every wave's), and every wave is past slab s-1, whose stage,
                // (s+3) % 4, takes slab s+3
                if (s + 2 < nslab)
                    wait_vmem<4>();
                else
                    wait_vmem<0>();
                lds_barrier();
                if (s + 3 < nslab) request(s + 3, Far());
            }
        }
    };
    int s0 = 0;
    for (; s0 + 4 <= nslab; s0 += 4) {
        slab(s0, I0(), acc[0], acc[1]);
        slab(s0 + 1, I1(), acc[1], acc[0]);
        slab(s0 + 2, I2(), acc[0], acc[1]);
        slab(s0 + 3, I3(), acc[1], acc[0]);
    }
    if (s0 < nslab) {   // nslab = 2 mod 4: two more, in stages 0 and 1
        slab(s0, I0(), acc[0], acc[1]);
        slab(s0 + 1, I1(), acc[1], acc[0]);
    }
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int i = 0; i < 16; ++i) accd[t][i] += (double)acc[1][t][i];

    const int L = qa.levels;
    const int64_t tile = (int64_t)rt * ncol + ct;
    uint32_t *tflags = qa.flags + tile * (BM * BN);
    const int lc = wc * 32 + l32;
    const int col = col0 + lc;
    // Code and flag of the lane's 32 outputs (one column, 32 rows).  thr(q)
    // is threshold q of this column before scaling by n.  The binary search
    // runs level by level over a tile's 16 outputs, so that their threshold
    // reads are independent (L is a power of two: c + step - 1 <= L - 2).
    auto epilogue = [&](auto thr) {
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            int c[16];
            double nr[16];
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                c[i] = 0;
                nr[i] = norm_s[wr * 64 + t * 32 + 8 * (i >> 2) + 4 * h + (i & 3)];
            }
            for (int step = L / 2; step >= 1; step >>= 1) {
#pragma unroll
                for (int i = 0; i < 16; ++i)
                    c[i] += (thr(c[i] + step - 1) * nr[i] <= accd[t][i]) ? step : 0;
            }
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int lr = wr * 64 + t * 32 + 8 * (i >> 2) + 4 * h + (i & 3);
                const int64_t gr = row0 + lr;
                const double y = accd[t][i];
                const double nrm = nr[i];
                const double tau = kTauRel * nrm + kTauAbs;
                const int ci = c[i];
                const double lo = thr(ci > 0 ? ci - 1 : 0) * nrm;
                const double hi = thr(ci < L - 1 ? ci : L - 2) * nrm;
                bool flag = !std::isfinite(y) || (ci > 0 && y - lo <= tau) ||
                            (ci < L - 1 && hi - y <= tau);
                int code = ci;
                if (nrm == 0.0) {
                    code = L / 2;
                    flag = false;
                }
                if (gr < m && col < d) {
                    qa.codes_tmp[gr * d + col] = (uint8_t)code;
                    if (flag) {
                        // a slot of this tile's list (an LDS counter)
                        const unsigned int slot = atomicAdd(&nflag_s, 1u);
                        tflags[slot] = ((uint32_t)lr << 7) | (uint32_t)lc;
                    }
                }
            }
        }
    };
    if (!qa.athr) {
        epilogue([&](int q) { return bnd_s[q]; });
    } else if (athr_lds) {
        epilogue([&](int q) { return athr_s[q * BN + lc]; });
    } else {
        const double *ac = qa.athr + (col < d ? col : d - 1);
        epilogue([&](int q) { return ac[(int64_t)q * d]; });
    }
    __syncthreads();
    if (tid == 0) qa.tile_count[tile] = nflag_s;
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

// Exact recomputation of flagged coordinates (b <= 4): the sequential
// float64 sum of the definition (products of float32 values are exact in
// float64, so fused and unfused multiply-adds agree).  One wave per output
// tile takes the tile's flags in batches of FX_FB, and for each slab of FX_KS
// coordinates every lane loads 16-byte pieces of the batch's X rows and R
// rows (one load instruction reads the 256-byte slabs of 4 flags' rows).
// The slabs are staged in LDS and lane f adds its flag's products in k
// order.  Two slabs are in registers while one is summed.
constexpr int FX_FB = 16;                    // flags per batch
constexpr int FX_KS = 64;                    // coordinates per slab (d is a multiple of 64)
constexpr int FX_PQ = FX_KS / 4;             // 16-byte pieces of a row slab
constexpr int FX_LD = FX_FB * FX_PQ / 64;    // load instructions per operand and slab

struct FxSlab {
    f4 x[FX_LD], r[FX_LD];
};

__global__ __launch_bounds__(64) void fixup_batch_kernel(
    const float *__restrict__ X, const float *__restrict__ R, int d, int ncol,
    const double *__restrict__ bounds, const double *__restrict__ athr, int levels,
    const double *__restrict__ norms,
    const uint32_t *__restrict__ flags, const unsigned int *__restrict__ tile_count,
    uint8_t *__restrict__ codes_tmp) {
    // flag f's slab at [f][FX_PQ + 1]: the padding puts the 16 summing
    // lanes' reads of one piece 17 pieces apart, in distinct banks
    constexpr int PS = FX_PQ + 1;
    __shared__ f4 xs[FX_FB * PS], rs[FX_FB * PS];
    const int tile = blockIdx.x;
    const int lane = threadIdx.x;
    const int64_t row0 = (int64_t)(tile / ncol) * BM;
    const int col0 = (tile % ncol) * BN;
    const int cnt = (int)tile_count[tile];
    const uint32_t *tflags = flags + (int64_t)tile * (BM * BN);
    const int ns = d / FX_KS;
    for (int e0 = 0; e0 < cnt; e0 += FX_FB) {
        const int nb = cnt - e0 < FX_FB ? cnt - e0 : FX_FB;
        // load i of a slab: lanes 16 g .. 16 g + 15 read the 256 contiguous
        // bytes of flag 4 i + g's row slab (piece lane mod 16)
        const float *xrow[FX_LD], *rrow[FX_LD];
#pragma unroll
        for (int i = 0; i < FX_LD; ++i) {
            const int f = 4 * i + (lane >> 4);
            const uint32_t fl = tflags[e0 + (f < nb ? f : nb - 1)];
            xrow[i] = X + (row0 + (fl >> 7)) * d + 4 * (lane & 15);
            rrow[i] = R + (int64_t)(col0 + (int)(fl & 127)) * d + 4 * (lane & 15);
        }
        const bool act = lane < nb;
        const uint32_t mf = tflags[e0 + (act ? lane : 0)];
        auto load = [&](int sl, FxSlab &b) {
#pragma unroll
            for (int i = 0; i < FX_LD; ++i) {
                b.x[i] = *reinterpret_cast<const f4 *>(xrow[i] + sl * FX_KS);
                b.r[i] = *reinterpret_cast<const f4 *>(rrow[i] + sl * FX_KS);
            }
        };
        // the barriers order the lanes' LDS accesses (a lane sums pieces
        // that other lanes staged): the previous slab's reads, the writes,
        // then the reads of the new slab; they leave the loads in flight
        auto stage = [&](const FxSlab &b) {
            lds_barrier();
#pragma unroll
            for (int i = 0; i < FX_LD; ++i) {
                const int at = (4 * i + (lane >> 4)) * PS + (lane & 15);
                xs[at] = b.x[i];
                rs[at] = b.r[i];
            }
            lds_barrier();
            // the refill of these registers stays after the writes: moved
            // ahead, it would take other registers and the loop would copy
            // them back at its back edge, waiting for every load in flight
            __builtin_amdgcn_sched_barrier(0);
        };
        double S = 0.0;
        auto sum = [&]() {
            if (act) {
#pragma unroll
                for (int q = 0; q < FX_PQ; ++q) {
                    const f4 a = rs[lane * PS + q];
                    const f4 b = xs[lane * PS + q];
#pragma unroll
                    for (int c = 0; c < 4; ++c) {
                        const double prod = (double)a[c] * (double)b[c];
                        S = S + prod;
                    }
                }
            }
        };
        // the loads are unconditional (clamped slab), so the waits count
        // them exactly
        FxSlab b0, b1;
        load(0, b0);
        __builtin_amdgcn_sched_barrier(0);   // b0's loads all ahead of b1's
        load(ns > 1 ? 1 : 0, b1);
        for (int sl = 0; sl < ns; sl += 2) {
            stage(b0);
            load(sl + 2 < ns ? sl + 2 : ns - 1, b0);
            sum();
            if (sl + 1 < ns) stage(b1);
            load(sl + 3 < ns ? sl + 3 : ns - 1, b1);
            if (sl + 1 < ns) sum();
        }
        if (act) {
            const int64_t row = row0 + (mf >> 7);
            const int j = col0 + (int)(mf & 127);
            codes_tmp[row * d + j] = (uint8_t)exact_code(S, norms[row], j, d, bounds, athr, levels);
        }
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

// Packs one row per thread, 64 rows per one-wave workgroup, for the bit
// widths whose 16-byte blocked chunk holds 128 / BITS codes as 4 words of
// 32 / BITS codes (BITS in {1, 2, 4, 8}; the canonical words are the same
// words): each lane walks its row's chunks in j order, adds fl64(c_code^2)
// (or the calibrated reconstruction's square) to the scale sum of the
// definition in j order, and writes the chunk's 16 bytes to the canonical
// and blocked layouts.  Every row of a chunk of rows is in flight at once,
// so the sequential sums (one dependent float64 add per code) overlap; the
// next chunk's codes are loaded while one is summed.
template <int BITS>
__global__ __launch_bounds__(64) void pack_rows_kernel(
    const uint8_t *__restrict__ codes_tmp, int64_t m, int d,
    const double *__restrict__ cent_sq, const double *__restrict__ ysq,
    const double *__restrict__ norms,
    uint8_t *__restrict__ canon, float *__restrict__ scales,
    uint8_t *__restrict__ blocked, float *__restrict__ blocked_scales, int64_t base,
    int chunks) {
    constexpr int L = 1 << BITS;
    constexpr int CPC = 128 / BITS;   // codes per chunk
    constexpr int LPC = CPC / 16;     // 16-byte loads of one-byte codes per chunk
    constexpr int PER = 32 / BITS;    // codes per word
    __shared__ double csq_s[L];
    const int lane = threadIdx.x;
    for (int i = lane; i < L; i += 64) csq_s[i] = ysq ? 0.0 : cent_sq[i];
    __syncthreads();
    const int64_t r = (int64_t)blockIdx.x * 64 + lane;
    if (r >= m) return;
    const uint4 *src = reinterpret_cast<const uint4 *>(codes_tmp + r * d);
    const int64_t v = base + r;
    uint8_t *bdst = blocked ? blocked + (v >> 6) * chunks * 1024 + (v & 63) * 16 : nullptr;
    uint8_t *cdst = canon ? canon + r * (int64_t)(d * BITS / 8) : nullptr;
    double h2 = 0.0;
    auto run = [&](auto cal_t) {
        constexpr bool CAL = decltype(cal_t)::value;
        uint4 cur[LPC], nxt[LPC];
#pragma unroll
        for (int i = 0; i < LPC; ++i) cur[i] = src[i];
        for (int ch = 0; ch < chunks; ++ch) {
            const int cn = ch + 1 < chunks ? ch + 1 : ch;
#pragma unroll
            for (int i = 0; i < LPC; ++i) nxt[i] = src[cn * LPC + i];
            uint32_t w[4] = {0u, 0u, 0u, 0u};
#pragma unroll
            for (int t = 0; t < CPC; ++t) {
                const uint4 &q = cur[t >> 4];
                const int u = (t >> 2) & 3;
                const uint32_t word = u == 0 ? q.x : u == 1 ? q.y : u == 2 ? q.z : q.w;
                const uint32_t code = (word >> (8 * (t & 3))) & 255u;
                w[t / PER] |= code << (BITS * (t % PER));
                double sq;
                if constexpr (CAL)
                    sq = ysq[(int64_t)(ch * CPC + t) * L + code];
                else
                    sq = csq_s[code];
                h2 = h2 + sq;
            }
            if (cdst) *reinterpret_cast<uint4 *>(cdst + ch * 16) = make_uint4(w[0], w[1], w[2], w[3]);
            if (bdst) {
                if (blocked_rotated(BITS))
                    for (int u = 0; u < 4; ++u) w[u] = rotl2(w[u]);
                *reinterpret_cast<uint4 *>(bdst + ch * 1024) = make_uint4(w[0], w[1], w[2], w[3]);
            }
#pragma unroll
            for (int i = 0; i < LPC; ++i) cur[i] = nxt[i];
        }
    };
    if (ysq)
        run(std::true_type{});
    else
        run(std::false_type{});
    const double nrm = norms[r];
    const float s = (nrm == 0.0) ? 0.0f : (float)(nrm / std::sqrt(h2));
    if (scales) scales[r] = s;
    if (blocked_scales) blocked_scales[base + r] = s;
}

// Packs PACK_ROWS rows per workgroup (3-bit codes): scale, canonical
// bitstream, blocked layout.
// The codes are staged in LDS with a row stride of d + 16 bytes, so that the
// scale threads (one per row, reading 16 codes at a time) meet different
// banks.
constexpr int PACK_ROWS = 32;   // PACK_ROWS * (d + 16) bytes of LDS (66 KiB at d = 2048)

__global__ __launch_bounds__(256) void pack_kernel(
    const uint8_t *__restrict__ codes_tmp, int64_t m, int d, int bits,
    const double *__restrict__ cent_sq, const double *__restrict__ ysq,
    const double *__restrict__ norms,
    uint8_t *__restrict__ canon, float *__restrict__ scales,
    uint8_t *__restrict__ blocked, float *__restrict__ blocked_scales, int64_t base,
    int chunks) {
    extern __shared__ __attribute__((aligned(16))) uint8_t cs_raw[];   // [PACK_ROWS][d + 16]
    __shared__ double csq_s[256];
    const int64_t r0 = (int64_t)blockIdx.x * PACK_ROWS;
    const int rows = (int)((m - r0) < PACK_ROWS ? (m - r0) : PACK_ROWS);
    const int tid = threadIdx.x;
    const int L = 1 << bits;
    const int ps = d + 16;           // LDS row stride
    if (!ysq)
        for (int i = tid; i < L; i += blockDim.x) csq_s[i] = cent_sq[i];
    // stage codes, 16 B per piece; each thread's pieces are loaded together
    const int vec_per_row = d / 16;
    const int total = rows * vec_per_row;
    constexpr int PIECES = PACK_ROWS * (2048 / 16) / 256;   // at most 16 per thread
    uint4 v[PIECES];
#pragma unroll
    for (int u = 0; u < PIECES; ++u) {
        const int e = min(tid + u * 256, total - 1);   // rows >= 1: a valid piece
        const int r = e / vec_per_row, q = e % vec_per_row;
        v[u] = reinterpret_cast<const uint4 *>(codes_tmp + (r0 + r) * d)[q];
    }
#pragma unroll
    for (int u = 0; u < PIECES; ++u) {
        const int e = tid + u * 256;
        if (e < total) {
            const int r = e / vec_per_row, q = e % vec_per_row;
            reinterpret_cast<uint4 *>(cs_raw + r * ps)[q] = v[u];
        }
    }
    __syncthreads();
    // scale: one thread per row, j in order
    if (tid < rows) {
        const uint8_t *c = cs_raw + tid * ps;
        // sum_j fl64(yhat_j^2): c[code]^2, or with TQ+ the calibrated
        // reconstruction's square, per coordinate ([d][levels])
        double h2 = 0.0;
        if (ysq) {
            for (int j = 0; j < d; ++j) h2 = h2 + ysq[(int64_t)j * L + c[j]];
        } else {
            for (int j = 0; j < d; j += 16) {
                const uint4 w = *reinterpret_cast<const uint4 *>(c + j);
#pragma unroll
                for (int q = 0; q < 4; ++q) h2 = h2 + csq_s[(w.x >> (8 * q)) & 255];
#pragma unroll
                for (int q = 0; q < 4; ++q) h2 = h2 + csq_s[(w.y >> (8 * q)) & 255];
#pragma unroll
                for (int q = 0; q < 4; ++q) h2 = h2 + csq_s[(w.z >> (8 * q)) & 255];
#pragma unroll
                for (int q = 0; q < 4; ++q) h2 = h2 + csq_s[(w.w >> (8 * q)) & 255];
            }
        }
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
            const uint8_t *c = cs_raw + r * ps;
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
            const uint8_t *c = cs_raw + r * ps;
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
// rot_gemm: every output element goes through the same
// v_mfma_f32_16x16x4f32 sequence per 32-wide slab (the same k in the same
// operand slots, sub and step order, from zero), the slab partials are
// folded into float64 in slab order and rounded to float32 at the end, so a
// row rotates to the same bits in either kernel.  The slab partials do not
// depend on each other, so they are computed in parallel: one workgroup per
// 16 x 16 output block, its 16 waves taking every 16th slab with all their
// loads issued at once; the partials meet in LDS and 256 threads fold them
// in order.  For short batches this is a few microseconds of latency (one
// round of loads) instead of 48 dependent slab steps.
constexpr int kSmallRows = 64;
constexpr int SPLIT_WAVES = 16;
constexpr int SPLIT_SLABS = 2048 / KB / SPLIT_WAVES;   // slabs per wave at most

__global__ __launch_bounds__(SPLIT_WAVES * 64) void rot_small_kernel(
    const float *__restrict__ X, int64_t m, int d, const float *__restrict__ R,
    float *__restrict__ Y, int *__restrict__ fill, int nfill, int fill_value) {
    __shared__ f4 part[2048 / KB][64];   // [slab][lane]: the 16 x 16 partial of a slab
    if (blockIdx.x == 0 && blockIdx.y == 0)
        for (int i = threadIdx.x; i < nfill; i += SPLIT_WAVES * 64) fill[i] = fill_value;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int l16 = lane & 15;
    const int g4 = lane >> 4;
    const int64_t r0 = (int64_t)blockIdx.y * 16;
    const int c0 = blockIdx.x * 16;
    const int64_t gr = r0 + l16;   // the row of X this lane loads
    const bool rowok = gr < m;
    const float *xa = X + (rowok ? gr : 0) * d + g4 * 4;
    const float *rb = R + (int64_t)(c0 + l16) * d + g4 * 4;
    const int nslab = d / KB;
    f4 fa[SPLIT_SLABS][2], fb[SPLIT_SLABS][2];
#pragma unroll
    for (int u = 0; u < SPLIT_SLABS; ++u) {
        const int s = wave + u * SPLIT_WAVES;
        if (s < nslab) {
#pragma unroll
            for (int sub = 0; sub < 2; ++sub) {
                fa[u][sub] = rowok ? *reinterpret_cast<const f4 *>(xa + s * KB + sub * 16)
                                   : f4{0.f, 0.f, 0.f, 0.f};
                fb[u][sub] = *reinterpret_cast<const f4 *>(rb + s * KB + sub * 16);
            }
        }
    }
#pragma unroll
    for (int u = 0; u < SPLIT_SLABS; ++u) {
        const int s = wave + u * SPLIT_WAVES;
        if (s < nslab) {
            f4 acc = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int sub = 0; sub < 2; ++sub)
#pragma unroll
                for (int st = 0; st < 4; ++st)
                    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[u][sub][st], fb[u][sub][st],
                                                               acc, 0, 0, 0);
            part[s][lane] = acc;
        }
    }
    __syncthreads();
    if (threadIdx.x < 256) {
        // output (row g4*4 + v, column l16) of the block: element v of lane (l16, g4)
        const int ln = threadIdx.x & 63;
        const int v = threadIdx.x >> 6;
        double accd = 0.0;
        for (int s = 0; s < nslab; ++s) accd += (double)part[s][ln][v];
        const int64_t row = r0 + (ln >> 4) * 4 + v;
        if (row < m) Y[row * d + c0 + (ln & 15)] = (float)accd;
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
        // one wave per 64 rows, spread over the CUs
        hipLaunchKernelGGL(row_norm_kernel, dim3((unsigned)((m + 63) / 64)), dim3(64), 0, stream,
                           X + r0 * d, m, d, norms, status_dev);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(encode_gemm, dim3(groups * 8 * ncol), dim3(GEMM_THREADS), 0,
                           stream, X + r0 * d, m, R, d, nrt, qa);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        // 8-bit codes flag about 2% of coordinates (thresholds ~4e-4 apart
        // at d = 1536): tiles then share their staged rows
        if (cb.levels > 16)
            hipLaunchKernelGGL(fixup_tile_kernel, dim3(nrt * ncol), dim3(GEMM_THREADS), 0, stream,
                               X + r0 * d, m, R, d, ncol, bounds, calib.athr, cb.levels, norms,
                               flags, tile_count, codes_tmp);
        else
            hipLaunchKernelGGL(fixup_batch_kernel, dim3(nrt * ncol), dim3(64), 0, stream, X + r0 * d,
                               R, d, ncol, bounds, calib.athr, cb.levels, norms, flags, tile_count,
                               codes_tmp);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        uint8_t *canon_p = out.canonical ? out.canonical + r0 * (int64_t)(d * cb.bits / 8) : nullptr;
        float *scales_p = out.scales ? out.scales + r0 : nullptr;
        const dim3 prow((unsigned)((m + 63) / 64));
        if (cb.bits == 3) {
            const int packs = (int)((m + PACK_ROWS - 1) / PACK_ROWS);
            hipLaunchKernelGGL(pack_kernel, dim3(packs), dim3(256), PACK_ROWS * (d + 16), stream,
                               codes_tmp, m, d, cb.bits, cent_sq, calib.ysq, norms, canon_p, scales_p,
                               out.blocked, out.blocked_scales, out.base + r0, chunks);
        } else if (cb.bits == 1) {
            hipLaunchKernelGGL(pack_rows_kernel<1>, prow, dim3(64), 0, stream, codes_tmp, m, d, cent_sq,
                               calib.ysq, norms, canon_p, scales_p, out.blocked, out.blocked_scales,
                               out.base + r0, chunks);
        } else if (cb.bits == 2) {
            hipLaunchKernelGGL(pack_rows_kernel<2>, prow, dim3(64), 0, stream, codes_tmp, m, d, cent_sq,
                               calib.ysq, norms, canon_p, scales_p, out.blocked, out.blocked_scales,
                               out.base + r0, chunks);
        } else if (cb.bits == 4) {
            hipLaunchKernelGGL(pack_rows_kernel<4>, prow, dim3(64), 0, stream, codes_tmp, m, d, cent_sq,
                               calib.ysq, norms, canon_p, scales_p, out.blocked, out.blocked_scales,
                               out.base + r0, chunks);
        } else {
            hipLaunchKernelGGL(pack_rows_kernel<8>, prow, dim3(64), 0, stream, codes_tmp, m, d, cent_sq,
                               calib.ysq, norms, canon_p, scales_p, out.blocked, out.blocked_scales,
                               out.base + r0, chunks);
        }
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

__global__ void fill_ints(int *p, int64_t n, int v) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

hipError_t rotate_rows_f32(const float *X, int64_t m, int d, const float *R, float *Y,
                           hipStream_t stream, int *fill, int64_t nfill, int fill_value) {
    if (!fill) nfill = 0;
    if (m > 0 && m <= kSmallRows && nfill <= kSmallRows) {
        const dim3 grid((unsigned)(d / 16), (unsigned)((m + 15) / 16));
        hipLaunchKernelGGL(rot_small_kernel, grid, dim3(SPLIT_WAVES * 64), 0, stream, X, m, d, R, Y,
                           fill, (int)nfill, fill_value);
        return hipGetLastError();
    }
    if (nfill > 0) {
        hipLaunchKernelGGL(fill_ints, dim3(1), dim3(256), 0, stream, fill, nfill, fill_value);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (m <= 0) return hipSuccess;
    const int ncol = (d + BN - 1) / BN;
    const int nrt = (int)((m + BM - 1) / BM);
    const int groups = (nrt + 7) / 8;
    hipLaunchKernelGGL(rot_gemm, dim3(groups * 8 * ncol), dim3(GEMM_THREADS), 0, stream, X, m, R,
                       d, nrt, Y);
    return hipGetLastError();
}

}  // namespace tq
