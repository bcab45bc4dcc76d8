// Wavefront-level top-k primitives on 64-lane waves (device code).
//
// A sorted list of 64*S entries lives in registers: rank r = 64*s + lane is
// held by `lane` in slot s.  The order is (score descending, id ascending);
// empty entries are (-inf, INT_MAX) and sort last.  Compare-exchange steps
// across lanes use cross-lane permutes; steps across slots stay in-lane.
#pragma once

#include <hip/hip_runtime.h>

#include <climits>
#include <cmath>

namespace tq {

struct Entry {
    float s;
    int i;
};

__device__ inline bool better(float sa, int ia, float sb, int ib) {
    return sa > sb || (sa == sb && ia < ib);
}

__device__ inline float shfl_xor_f(float v, int m) { return __shfl_xor(v, m, 64); }
__device__ inline int shfl_xor_i(int v, int m) { return __shfl_xor(v, m, 64); }
__device__ inline float shfl_f(float v, int src) { return __shfl(v, src, 64); }
__device__ inline int shfl_i(int v, int src) { return __shfl(v, src, 64); }

// Bitonic sort of one entry per lane into descending order.
__device__ inline void wave_sort64(float &s, int &i, int lane) {
#pragma unroll
    for (int k = 2; k <= 64; k <<= 1) {
#pragma unroll
        for (int j = k >> 1; j > 0; j >>= 1) {
            const float os = shfl_xor_f(s, j);
            const int oi = shfl_xor_i(i, j);
            const bool lower = (lane & j) == 0;
            const bool desc = (lane & k) == 0;
            const bool ob = better(os, oi, s, i);
            if ((lower == desc) ? ob : !ob) {
                s = os;
                i = oi;
            }
        }
    }
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
    for (int j = 32; j > 0; j >>= 1) {
        const bool lower = (lane & j) == 0;
#pragma unroll
        for (int a = 0; a < S; ++a) {
            const float os = shfl_xor_f(s[a], j);
            const int oi = shfl_xor_i(i[a], j);
            const bool ob = better(os, oi, s[a], i[a]);
            if (lower ? ob : !ob) {
                s[a] = os;
                i[a] = oi;
            }
        }
    }
}

// list <- top 64*S of (list U new), `new` being one sorted (descending) entry
// per lane.
template <int S>
__device__ inline void merge_sorted64(float (&ls)[S], int (&li)[S], float ns, int ni, int lane) {
    const float rs = shfl_f(ns, 63 - lane);
    const int ri = shfl_i(ni, 63 - lane);
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
        const float rs = shfl_f(os[S - 1 - a], 63 - lane);
        const int ri = shfl_i(oi[S - 1 - a], 63 - lane);
        if (better(rs, ri, ls[a], li[a])) {
            ls[a] = rs;
            li[a] = ri;
        }
    }
    bitonic_merge<S>(ls, li, lane);
}

// Value of rank r (uniform) of a list.
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
    s = shfl_f(vs, ln);
    i = shfl_i(vi, ln);
}

}  // namespace tq
