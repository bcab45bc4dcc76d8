// Wavefront-level top-k primitives on 64-lane waves (device code).
//
// A sorted list of 64*S entries lives in registers: rank r = 64*s + lane is
// held by `lane` in slot s.  The order is (score descending, id ascending);
// empty entries are (-inf, INT_MAX) and sort last.
//
// Sorting network: bitonic sort in its "flip" form -- for block size k the
// first stage compares lane i with its mirror i ^ (k-1), the following
// half-cleaner stages compare i with i ^ j for j = k/4 .. 1, and every
// comparison keeps the better entry at the lower lane, so no direction bits
// are needed.  Partners within a row of 16 lanes are reached with DPP lane
// permutations (quad_perm, row_half_mirror, row_mirror, row_ror) on the
// vector ALU; only partners 16, 31, 32 and 63 lanes away use a cross-lane
// permute through the LDS crossbar.
#pragma once

#include <hip/hip_runtime.h>

#include <climits>
#include <cmath>

namespace tq {

__device__ inline bool better(float sa, int ia, float sb, int ib) {
    return sa > sb || (sa == sb && ia < ib);
}

// DPP control codes (GFX9 encoding).
constexpr int kDppXor1 = 0xB1;        // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;        // quad_perm [2,3,0,1]
constexpr int kDppXor3 = 0x1B;        // quad_perm [3,2,1,0]
constexpr int kDppRowShl4 = 0x104;    // lane i <- lane i+4 within the row
constexpr int kDppRowShr4 = 0x114;    // lane i <- lane i-4 within the row
constexpr int kDppRowRor8 = 0x128;    // lane i <- lane (i+8) mod 16 == i ^ 8
constexpr int kDppRowRor4 = 0x124;    // lane i <- lane (i+4) mod 16 within the row
constexpr int kDppRowRor2 = 0x122;    // lane i <- lane (i+2) mod 16
constexpr int kDppRowRor1 = 0x121;    // lane i <- lane (i+1) mod 16
constexpr int kDppRowMirror = 0x140;  // lane i <- lane 15-i == i ^ 15
constexpr int kDppHalfMirror = 0x141; // lane i <- lane 7-i within 8 == i ^ 7

template <int CTRL>
__device__ inline int dpp_i(int v) {
    return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, false);
}
template <int CTRL>
__device__ inline float dpp_f(float v) {
    return __int_as_float(dpp_i<CTRL>(__float_as_int(v)));
}

// Value held by lane (lane ^ M).
template <int M>
__device__ inline int xor_i(int v, int lane) {
    if constexpr (M == 1) return dpp_i<kDppXor1>(v);
    else if constexpr (M == 2) return dpp_i<kDppXor2>(v);
    else if constexpr (M == 3) return dpp_i<kDppXor3>(v);
    else if constexpr (M == 4) {
        const int up = dpp_i<kDppRowShl4>(v);
        const int dn = dpp_i<kDppRowShr4>(v);
        return (lane & 4) ? dn : up;
    } else if constexpr (M == 7) return dpp_i<kDppHalfMirror>(v);
    else if constexpr (M == 8) return dpp_i<kDppRowRor8>(v);
    else if constexpr (M == 15) return dpp_i<kDppRowMirror>(v);
    else return __shfl_xor(v, M, 64);
}
template <int M>
__device__ inline float xor_f(float v, int lane) {
    return __int_as_float(xor_i<M>(__float_as_int(v), lane));
}

// Compare-exchange of lane i with lane i ^ M; the lane whose bit LB is clear
// keeps the better entry.
template <int M, int LB>
__device__ inline void cx(float &s, int &i, int lane) {
    const float os = xor_f<M>(s, lane);
    const int oi = xor_i<M>(i, lane);
    const bool lower = (lane & LB) == 0;
    const bool ob = better(os, oi, s, i);
    if (lower == ob) {
        s = os;
        i = oi;
    }
}

// Half-cleaner stages j = J, J/2, .. 1 on one register.
template <int J>
__device__ inline void half_clean(float &s, int &i, int lane) {
    if constexpr (J >= 1) {
        cx<J, J>(s, i, lane);
        half_clean<J / 2>(s, i, lane);
    }
}

// Bitonic sort of one entry per lane into descending order.
__device__ inline void wave_sort64(float &s, int &i, int lane) {
    cx<1, 1>(s, i, lane);
    cx<3, 2>(s, i, lane);
    half_clean<1>(s, i, lane);
    cx<7, 4>(s, i, lane);
    half_clean<2>(s, i, lane);
    cx<15, 8>(s, i, lane);
    half_clean<4>(s, i, lane);
    cx<31, 16>(s, i, lane);
    half_clean<8>(s, i, lane);
    cx<63, 32>(s, i, lane);
    half_clean<16>(s, i, lane);
}

// Half-cleaner stages of a bitonic merge over 64*S entries (S slots), leaving
// them in descending order.
template <int S>
__device__ inline void bitonic_merge(float (&s)[S], int (&i)[S], int lane) {
#pragma unroll
    for (int j = 32 * S; j >= 64; j >>= 1) {
        const int js = j / 64;
#pragma unroll
        for (int a = 0; a < S; ++a) {
            if ((a & js) == 0) {
                const int b = a + js;
                if (better(s[b], i[b], s[a], i[a])) {
                    const float ts = s[a];
                    const int ti = i[a];
                    s[a] = s[b];
                    i[a] = i[b];
                    s[b] = ts;
                    i[b] = ti;
                }
            }
        }
    }
#pragma unroll
    for (int a = 0; a < S; ++a) half_clean<32>(s[a], i[a], lane);
}

// list <- top 64*S of (list U new), `new` being one sorted (descending) entry
// per lane.
template <int S>
__device__ inline void merge_sorted64(float (&ls)[S], int (&li)[S], float ns, int ni, int lane) {
    const float rs = xor_f<63>(ns, lane);     // new list reversed
    const int ri = xor_i<63>(ni, lane);
    if (better(rs, ri, ls[S - 1], li[S - 1])) {
        ls[S - 1] = rs;
        li[S - 1] = ri;
    }
    bitonic_merge<S>(ls, li, lane);
}

// list <- top 64*S of (list U other), both sorted lists of 64*S entries.
template <int S>
__device__ inline void merge_lists(float (&ls)[S], int (&li)[S], const float (&os)[S],
                                   const int (&oi)[S], int lane) {
#pragma unroll
    for (int a = 0; a < S; ++a) {
        // rank 64a + lane of list meets rank 64S-1-(64a+lane) of other
        const float rs = xor_f<63>(os[S - 1 - a], lane);
        const int ri = xor_i<63>(oi[S - 1 - a], lane);
        if (better(rs, ri, ls[a], li[a])) {
            ls[a] = rs;
            li[a] = ri;
        }
    }
    bitonic_merge<S>(ls, li, lane);
}

// Value of rank r (wave-uniform) of a list, returned wave-uniform.
template <int S>
__device__ inline void rank_entry(const float (&ls)[S], const int (&li)[S], int r, float &s,
                                  int &i) {
    const int slot = r >> 6, ln = r & 63;
    float vs = ls[0];
    int vi = li[0];
#pragma unroll
    for (int a = 1; a < S; ++a)
        if (slot == a) {
            vs = ls[a];
            vi = li[a];
        }
    s = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(vs), ln));
    i = __builtin_amdgcn_readlane(vi, ln);
}

// Order-preserving map of float32 onto int32 (for atomicMax thresholds).
__device__ inline int fkey(float f) {
    const int b = __float_as_int(f);
    return b >= 0 ? b : (b ^ 0x7FFFFFFF);
}
__device__ inline float unfkey(int k) { return __int_as_float(k >= 0 ? k : (k ^ 0x7FFFFFFF)); }

// A wave's best 64*S (score, id) entries, kept sorted in registers, with
// the k-th best as threshold.
template <int S>
struct WaveTopK {
    float ls[S];
    int li[S];
    float th_s;      // this wave's k-th best (or -inf while fewer than k)
    int th_i;
    int seen_g;      // last global bound read (order key)
    __device__ void reset() {
#pragma unroll
        for (int a = 0; a < S; ++a) {
            ls[a] = -INFINITY;
            li[a] = INT_MAX;
        }
        th_s = -INFINITY;
        th_i = INT_MAX;
        seen_g = fkey(-INFINITY);
    }
    // Offer one (score, id) per lane.  A score strictly below the bound --
    // the best k-th score any wave of this workgroup (wg_key, LDS) or of any
    // workgroup (g_key, global) has proven -- cannot reach the top k and is
    // dropped before the sort.
    __device__ void offer(float sc, int id, int lane, int k, int *wg_key, int *g_key) {
        offer_seen(sc, id, lane, k, wg_key, g_key,
                   __hip_atomic_load(g_key, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
    }
    // As offer(), with gk a value of the global bound read earlier by the
    // caller (any earlier value is a valid, if weaker, bound).
    __device__ void offer_seen(float sc, int id, int lane, int k, int *wg_key, int *g_key, int gk) {
        seen_g = gk > seen_g ? gk : seen_g;
        const int bk = *wg_key > seen_g ? *wg_key : seen_g;
        const float bound = unfkey(bk);
        const bool cand = better(sc, id, th_s, th_i) && !(sc < bound);
        if (__any(cand)) {
            if (!cand) {
                sc = -INFINITY;
                id = INT_MAX;
            }
            wave_sort64(sc, id, lane);
            merge_sorted64<S>(ls, li, sc, id, lane);
            rank_entry<S>(ls, li, k - 1, th_s, th_i);
            if (th_s > -INFINITY) {
                const int key = fkey(th_s);
                if (lane == 0) atomicMax(wg_key, key);
                if (key > seen_g) {
                    if (lane == 0)
                        __hip_atomic_fetch_max(g_key, key, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    seen_g = key;
                }
            }
        }
    }
};

}  // namespace tq
