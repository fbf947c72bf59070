// Device helpers shared by the kernels of libsnn (gfx950, wave64).
#pragma once

#include "snn_internal.h"

extern __shared__ __align__(16) unsigned char smem[];

namespace {

extern __shared__ __align__(16) unsigned char smem[];

__device__ __forceinline__ unsigned long long uniform64(unsigned long long x) {
    const unsigned lo = __builtin_amdgcn_readfirstlane((unsigned)x);
    const unsigned hi = __builtin_amdgcn_readfirstlane((unsigned)(x >> 32));
    return ((unsigned long long)hi << 32) | lo;
}

__device__ __forceinline__ int uniform32(int x) { return __builtin_amdgcn_readfirstlane(x); }

// number of set bits of m in lanes below this one
__device__ __forceinline__ int lanes_below(unsigned long long m) {
    return (int)__builtin_amdgcn_mbcnt_hi((unsigned)(m >> 32),
                                          __builtin_amdgcn_mbcnt_lo((unsigned)m, 0u));
}

// Pointers typed with their address space: LDS and global accesses are never
// folded into one flat access, and the fp64 LDS atomic is ds_add_f64.
typedef __attribute__((address_space(3))) double lds_f64;
typedef __attribute__((address_space(1))) float global_f32;
typedef __attribute__((address_space(3))) float lds_f32;

__device__ __forceinline__ void lds_add_f64(double* p, double v) {
    __hip_atomic_fetch_add((lds_f64*)p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// x of the lane given by the DPP control CTRL (within 16-lane rows), fp64 as
// two 32-bit moves.
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double x) {
    const unsigned long long u = (unsigned long long)__double_as_longlong(x);
    const int lo = __builtin_amdgcn_update_dpp(0, (int)(unsigned)u, CTRL, 0xF, 0xF, false);
    const int hi = __builtin_amdgcn_update_dpp(0, (int)(unsigned)(u >> 32), CTRL, 0xF, 0xF, false);
    return __longlong_as_double((long long)(((unsigned long long)(unsigned)hi << 32) | (unsigned)lo));
}

__device__ __forceinline__ double read_lane_f64(double x, int lane) {
    const unsigned long long u = (unsigned long long)__double_as_longlong(x);
    const unsigned lo = __builtin_amdgcn_readlane((int)(unsigned)u, lane);
    const unsigned hi = __builtin_amdgcn_readlane((int)(unsigned)(u >> 32), lane);
    return __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
}

// Sum of x over the 64 lanes of a fully active wave, uniform.  Within each
// 16-lane row: quad_perm [1,0,3,2], quad_perm [2,3,0,1], half-row mirror and
// row mirror leave the row sum in every lane; the four row sums are read out
// and added.
__device__ __forceinline__ double wave_sum(double x) {
    x += dpp_f64<0xB1>(x);
    x += dpp_f64<0x4E>(x);
    x += dpp_f64<0x141>(x);
    x += dpp_f64<0x140>(x);
    return (read_lane_f64(x, 0) + read_lane_f64(x, 16)) + (read_lane_f64(x, 32) + read_lane_f64(x, 48));
}

inline unsigned grid_for(long long n, int block) { return (unsigned)((n + block - 1) / block); }

// ------------------------------------------------------------------ batched ring updates

constexpr int KB = 8;   // spikes per batch

// Adds w[k] to the cells row[k] (row < 0: skip) of one lane's ring column
// (cell r at col[r * stride]) in the order k = 0 .. KB-1.  All reads are
// issued first, equal rows are merged in registers (the later update starts
// from the earlier one's result), then the writes go out in order: the fp32
// result equals one read-modify-write per spike in order.
template <typename Ptr>
__device__ __forceinline__ void column_add(Ptr col, int stride, const int (&row)[KB],
                                           const float (&w)[KB]) {
    float v[KB];
#pragma unroll
    for (int k = 0; k < KB; ++k) v[k] = (row[k] >= 0) ? col[row[k] * stride] : 0.0f;
#pragma unroll
    for (int k = 0; k < KB; ++k) {
        float base = v[k];
#pragma unroll
        for (int j = 0; j < k; ++j) base = (row[j] == row[k]) ? v[j] : base;
        v[k] = __fadd_rn(base, w[k]);
    }
#pragma unroll
    for (int k = 0; k < KB; ++k)
        if (row[k] >= 0) col[row[k] * stride] = v[k];
}

// Up to KB consecutive entries of a uniform index list; -1 past the end.
__device__ __forceinline__ void list_chunk(const int* list, int k0, int k_hi, int (&ids)[KB]) {
#pragma unroll
    for (int k = 0; k < KB; ++k) ids[k] = (k0 + k < k_hi) ? uniform32(list[k0 + k]) : -1;
}

// Weights and ring rows of a chunk of presynaptic spikes at step n for post
// column j of a projection (weights W, slots Sp, nq posts).
__device__ __forceinline__ void chunk_rows(const float* W, const uint8_t* Sp, int nq, int j, int n,
                                           int n_mod, int S, int T, const int (&ids)[KB],
                                           int (&row)[KB], float (&w)[KB]) {
#pragma unroll
    for (int k = 0; k < KB; ++k) {
        row[k] = -1;
        w[k] = 0.0f;
        if (ids[k] >= 0) {
            const size_t kk = (size_t)ids[k] * nq + j;
            const int s = Sp[kk];
            w[k] = W[kk];
            if (n + s <= T - 1) {
                const int r = n_mod + s;
                row[k] = (r >= S) ? r - S : r;
            }
        }
    }
}

// ------------------------------------------------------------------ forward core

// Set bits of nw ballot masks in LDS, ascending.
struct BitIter {
    const unsigned long long* mk;
    int nw, w;
    unsigned long long cur;
};

__device__ __forceinline__ BitIter bits_begin(const unsigned long long* mk, int nw) {
    BitIter it;
    it.mk = mk;
    it.nw = nw;
    it.w = 0;
    it.cur = uniform64(mk[0]);
    return it;
}

template <int N>
__device__ __forceinline__ bool bits_chunk(BitIter& it, int (&ids)[N]) {
    bool any = false;
#pragma unroll
    for (int k = 0; k < N; ++k) {
        while (it.cur == 0 && it.w + 1 < it.nw) it.cur = uniform64(it.mk[++it.w]);
        if (it.cur) {
            ids[k] = it.w * 64 + __builtin_ctzll(it.cur);
            it.cur &= it.cur - 1;
            any = true;
        } else {
            ids[k] = -1;
        }
    }
    return any;
}

}  // namespace
