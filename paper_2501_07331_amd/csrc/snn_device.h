// Device helpers shared by the kernels of libsnn (gfx950, wave64).
#pragma once

#include <type_traits>

#include "snn_internal.h"

// dynamic LDS of every kernel
extern __shared__ __align__(16) unsigned char smem[];

namespace {

__device__ __forceinline__ unsigned long long uniform64(unsigned long long x) {
    const unsigned lo = __builtin_amdgcn_readfirstlane((unsigned)x);
    const unsigned hi = __builtin_amdgcn_readfirstlane((unsigned)(x >> 32));
    return ((unsigned long long)hi << 32) | lo;
}


// number of set bits of m in lanes below this one
__device__ __forceinline__ int lanes_below(unsigned long long m) {
    return (int)__builtin_amdgcn_mbcnt_hi((unsigned)(m >> 32),
                                          __builtin_amdgcn_mbcnt_lo((unsigned)m, 0u));
}

// Pointers typed with their address space: LDS and global accesses are never
// folded into one flat access, and the fp64 LDS atomic is ds_add_f64.
typedef __attribute__((address_space(1))) float global_f32;
typedef __attribute__((address_space(3))) float lds_f32;
typedef __attribute__((address_space(1))) double global_f64;
typedef __attribute__((address_space(3))) double lds_f64;
// destination of a direct load into LDS (wave-uniform base; lane k's data
// lands at base + k * size)
typedef __attribute__((address_space(3))) void* lds_ptr_t;
// A device-memory pointer typed as such.  Pointers that a kernel keeps in
// vector registers (made opaque by an empty asm) need it: a generic pointer
// there loses its address space, and its accesses become flat ones, which
// also count on the LDS counter, so that every later wait for an LDS access
// waits for them too.
template <typename T>
using gptr = __attribute__((address_space(1))) T*;

// x of the lane given by the DPP control CTRL (within 16-lane rows), fp64 as
// two 32-bit moves.
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double x) {
    const unsigned long long u = (unsigned long long)__double_as_longlong(x);
    const int lo = __builtin_amdgcn_update_dpp(0, (int)(unsigned)u, CTRL, 0xF, 0xF, false);
    const int hi = __builtin_amdgcn_update_dpp(0, (int)(unsigned)(u >> 32), CTRL, 0xF, 0xF, false);
    return __longlong_as_double((long long)(((unsigned long long)(unsigned)hi << 32) | (unsigned)lo));
}

inline unsigned grid_for(long long n, int block) { return (unsigned)((n + block - 1) / block); }

// spikes per chunk of the delayed scatters
constexpr int KB = 8;

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

// The words of a spike-mask row, uniform (NWM >= NW words; the rest zero).
template <int NWM>
__device__ __forceinline__ void row_words(const unsigned long long* row, int NW,
                                          unsigned long long (&m)[NWM]) {
    // every read stays in the row (no branch around it); words past NW are
    // zeroed after the read
#pragma unroll
    for (int w = 0; w < NWM; ++w) {
        const unsigned long long v = row[min(w, NW - 1)];
        m[w] = (w < NW) ? v : 0ull;
    }
#pragma unroll
    for (int w = 0; w < NWM; ++w) m[w] = uniform64(m[w]);
}

// Position of set bit number r (0-based, r < popcount) of a 64-bit word, by
// halving: branch-free, per lane.
__device__ __forceinline__ int nth_bit(unsigned long long word, int r) {
    const unsigned lo = (unsigned)word, hi = (unsigned)(word >> 32);
    int c = __popc(lo);
    bool up = r >= c;
    r -= up ? c : 0;
    unsigned x = up ? hi : lo;
    int pos = up ? 32 : 0;
#pragma unroll
    for (int h = 16; h >= 2; h >>= 1) {
        const unsigned low = x & ((1u << h) - 1u);
        c = __popc(low);
        up = r >= c;
        r -= up ? c : 0;
        x = up ? (x >> h) : low;
        pos += up ? h : 0;
    }
    return pos + ((r >= (int)(x & 1u)) ? 1 : 0);
}

// Set bits of a spike-mask row, ascending: skip the first `skip`, return the
// next N (-1 past the end), uniform.  Up to four words (m: the row's words,
// uniform), or any number with LP, lane q finds set bit number skip + q
// branch-free and the ids are read from lanes 0 .. N-1; longer rows (row: the
// same NW words in LDS) are otherwise walked word by word at run time, which
// keeps the code small but puts an LDS round trip on every word (LP suits a
// lone wave, whose every LDS latency is exposed).
template <int NWM, int N, bool LP = false>
__device__ __forceinline__ void word_ids(const unsigned long long (&m)[NWM],
                                         const unsigned long long* row, int NW, int skip,
                                         int (&ids)[N]) {
    static_assert(N <= 64, "one lane per id");
    if constexpr (NWM > 4 && !LP) {
        BitIter it = bits_begin(row, NW);
        for (;;) {
            const int c = __popcll(it.cur);
            if (c > skip || it.w + 1 >= NW) break;
            skip -= c;
            it.cur = uniform64(row[++it.w]);
        }
        for (; skip > 0 && it.cur; --skip) it.cur &= it.cur - 1;
        bits_chunk<N>(it, ids);
    } else {
        const int q = (int)(threadIdx.x & 63) + skip;
        int base = 0, wsel = -1, bsel = 0;
        unsigned long long word = 0;
#pragma unroll
        for (int w = 0; w < NWM; ++w) {
            const int c = __popcll(m[w]);
            const bool here = wsel < 0 && q < base + c;
            word = here ? m[w] : word;
            bsel = here ? base : bsel;
            wsel = here ? w : wsel;
            base += c;
        }
        const int id = (wsel < 0) ? -1 : wsel * 64 + nth_bit(word, q - bsel);
#pragma unroll
        for (int k = 0; k < N; ++k) ids[k] = __builtin_amdgcn_readlane(id, k);
    }
}

// s_waitcnt vmcnt(0), expcnt and lgkmcnt left at their maximum (gfx9 encoding)
constexpr int kWaitVm0 = 0x0F70;

// ------------------------------------------------------------------ cluster exchange

// Cluster and rank of workgroup k of a cluster launch (G workgroups per
// cluster).  Workgroups are dealt to the 8 XCDs round robin (k mod 8), so
// when G is a multiple of 8 the ranks are dealt the same way: every XCD
// serves G / 8 ranks, i.e. the same column slices of every weight matrix in
// all clusters, which its L2 keeps.  Any other G: consecutive workgroups.
// Either way a bijection onto (cluster, rank).
__device__ __forceinline__ void cluster_rank(int k, int G, int& c, int& g) {
    if (G % 8 == 0) {
        const int per = G / 8, i = k / 8;
        g = (k % 8) * per + i % per;
        c = i / per;
    } else {
        c = k / G;
        g = k % G;
    }
}

// Polls after which a cluster wait gives up (a poll is one device-memory
// round trip of about a microsecond, so about two seconds): the wave then
// raises the abort flag and its kernel returns; every other wait of the
// launch sees the flag within 256 polls and returns too.
constexpr int kClusterSpins = 1 << 21;

// Word p <- (tag, payload), one agent-scope atomic store.
__device__ __forceinline__ void cl_put(unsigned long long* p, unsigned tag, unsigned payload) {
    __hip_atomic_store(p, ((unsigned long long)tag << 32) | payload, __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
}

// Every lane with want waits until word X[k] carries tag and takes its
// payload (the wave polls until all of them have); all 64 lanes call it.
// false: the wait gave up or another wave did (the abort flag is set).
__device__ __forceinline__ bool cl_get(const unsigned long long* X, int k, bool want, unsigned tag,
                                      unsigned& v, int* abort_flag) {
    bool ok = !want;
    unsigned long long w = 0;
    for (int spin = 0;; ++spin) {
        if (!ok) {
            w = __hip_atomic_load(X + k, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            ok = (unsigned)(w >> 32) == tag;
        }
        if (__ballot(!ok) == 0) break;
        if ((spin & 255) == 255) {
            if (__hip_atomic_load(abort_flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) return false;
            if (spin >= kClusterSpins) {
                __hip_atomic_store(abort_flag, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                return false;
            }
        }
        __builtin_amdgcn_s_sleep(1);
    }
    v = (unsigned)w;
    return true;
}

// One leaky-integrator neuron (a LIF neuron without threshold).
struct LiState {
    float V, I, acc, best;
    int nst;
};

// One LI step n: V- = fma(alpha, V, gamma I), I- = beta I, the readout
// statistic of V- (running sum, or first maximum and its step), then the
// step's arrivals x added to I.
template <bool SUM>
__device__ __forceinline__ void li_update(float alpha, float beta, float gamma, int n, float x,
                                          LiState& q) {
    const float gi = __fmul_rn(gamma, q.I);
    const float Vm = __fmaf_rn(alpha, q.V, gi);
    q.I = __fmul_rn(beta, q.I);
    q.V = Vm;
    if (SUM) {
        q.acc = __fadd_rn(q.acc, Vm);
    } else if (n == 0 || Vm > q.best) {
        q.best = Vm;
        q.nst = n;
    }
    q.I = __fadd_rn(q.I, x);
}

// Adds w[k] to cell row[k] of one lane's column (cell r at col[r * stride])
// for k = 0 .. K-1 in order, where every row is valid (out-of-range entries
// point at a dummy row that is never read out).  Reads first, equal rows
// merged in registers, then the writes: the same fp32 result as one
// read-modify-write per entry in order, without branches.
template <typename Ptr, int K>
__device__ __forceinline__ void column_add_all(Ptr col, int stride, const int (&row)[K],
                                               const float (&w)[K]) {
    float v[K];
#pragma unroll
    for (int k = 0; k < K; ++k) v[k] = col[row[k] * stride];
#pragma unroll
    for (int k = 0; k < K; ++k) {
        float base = v[k];
#pragma unroll
        for (int j = 0; j < k; ++j) base = (row[j] == row[k]) ? v[j] : base;
        v[k] = __fadd_rn(base, w[k]);
    }
#pragma unroll
    for (int k = 0; k < K; ++k) col[row[k] * stride] = v[k];
}

// The same sums for a column in LDS, in rounds of P entries: a round reads
// its P cells, merges equal rows among them in registers, adds and writes
// back, and the next round's reads are issued after those writes (the LDS
// accesses of a lane complete in order), so they see them.  Fewer merge
// instructions (P (P - 1) / 2 pairs per round instead of K (K - 1) / 2) for
// more LDS round trips; P = 2 is the fastest split for chunks of 8 on gfx950.
template <int P, int K>
__device__ __forceinline__ void column_add_rounds(lds_f32* col, int stride, const int (&row)[K],
                                                  const float (&w)[K]) {
    static_assert(K % P == 0, "rounds must cover the chunk");
#pragma unroll
    for (int h = 0; h < K / P; ++h) {
        float v[P];
#pragma unroll
        for (int k = 0; k < P; ++k) v[k] = col[row[h * P + k] * stride];
#pragma unroll
        for (int k = 0; k < P; ++k) {
            float base = v[k];
#pragma unroll
            for (int j = 0; j < k; ++j) base = (row[h * P + j] == row[h * P + k]) ? v[j] : base;
            v[k] = __fadd_rn(base, w[h * P + k]);
        }
#pragma unroll
        for (int k = 0; k < P; ++k) col[row[h * P + k] * stride] = v[k];
    }
}

// Chunk sums into a column: in LDS in rounds of two entries, in device
// memory all at once (every round there would be a memory round trip).
template <typename Ptr, int K>
__device__ __forceinline__ void column_add(Ptr col, int stride, const int (&row)[K], const float (&w)[K]) {
    if constexpr (std::is_same<Ptr, lds_f32*>::value)
        column_add_rounds<2>(col, stride, row, w);
    else
        column_add_all(col, stride, row, w);
}

// Delayed scatter of a sorted event list into a table, one column per lane:
// for every event e in [e_lo, e_hi) in order (presynaptic neuron ids[e] at
// step steps[e]), the lane adds w(ids[e], col) to the cell of arrival step
// m = steps[e] + slot(ids[e], col) when m lies in [m0, m_end): cell
// tab[(m - m0) * ld] of the lane's column; everything else goes to the dummy
// row `dummy` (>= m_end - m0) of the column.  ws holds (weight bits, slot)
// rows of npost entries (ws_bytes in all, the bound of the buffer loads);
// lanes with live == false add to the dummy row only.
//
// Chunks of KB events, software-pipelined in pairs: while a chunk is added,
// the weight rows of the next chunk and the ids and steps of the next pair
// of chunks (one event per lane) are in flight.  One wait at each chunk
// start covers the loads issued a chunk earlier, and the weight registers
// alternate between the two chunks of a pair, so no register copy waits for
// a load in flight.  A lane adds a chunk to its own column in event order
// (column_add: in LDS in rounds of two events; fp32 LDS atomics would keep
// the order too, but are far slower).
template <typename Ptr>
__device__ __forceinline__ void scatter_events(const int* ids, const int* steps, int e_lo, int e_hi,
                                               const uint2* ws, int ws_bytes, int npost, int col,
                                               bool live, int m0, int m_end, int dummy, Ptr tab,
                                               int ld) {
    if (e_hi <= e_lo) return;
    const int lane = threadIdx.x & 63;
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc((void*)ws, (short)0, ws_bytes,
                                                                        0x00020000);
    const int col8 = min(max(col, 0), npost - 1) * 8;
    const int row8 = npost * 8;
    const unsigned span = (unsigned)(live ? m_end - m0 : 0);   // dead lanes: all to the dummy
    // lane q < 2 KB: event e0 + q, the byte offset of its weight row and its step
    auto load_pair = [&](int e0, int& id, int& st) {
        const int e = min(e0 + (lane & (2 * KB - 1)), e_hi - 1);
        id = ids[e] * row8;
        st = steps[e];
    };
    auto load_ws = [&](int off_v, int qoff, uint2 (&w)[KB]) {
#pragma unroll
        for (int q = 0; q < KB; ++q) {
            const int off = __builtin_amdgcn_readlane(off_v, qoff + q);
            const auto v = __builtin_amdgcn_raw_buffer_load_b64(rs, col8, off, 0);
            w[q] = make_uint2((unsigned)v[0], (unsigned)v[1]);
        }
    };
    auto add = [&](int e0, int st_v, int qoff, const uint2 (&w)[KB]) {
        const int nv = e_hi - e0;                      // valid events from e0 on (uniform)
        int row[KB];
        float wv[KB];
#pragma unroll
        for (int q = 0; q < KB; ++q) {
            const int d = __builtin_amdgcn_readlane(st_v, qoff + q) + (int)w[q].y - m0;
            row[q] = (q < nv && (unsigned)d < span) ? d : dummy;
            wv[q] = __uint_as_float(w[q].x);
        }
        column_add(tab, ld, row, wv);
    };
    int idA, stA, idB, stB;
    uint2 w0[KB], w1[KB];
    load_pair(e_lo, idA, stA);
    __builtin_amdgcn_s_waitcnt(kWaitVm0);
    load_ws(idA, 0, w0);
    for (int e0 = e_lo; e0 < e_hi; e0 += 2 * KB) {
        __builtin_amdgcn_s_waitcnt(kWaitVm0);
        load_pair(e0 + 2 * KB, idB, stB);
        load_ws(idA, KB, w1);                          // second chunk of this pair
        add(e0, stA, 0, w0);
        if (e0 + KB >= e_hi) break;
        __builtin_amdgcn_s_waitcnt(kWaitVm0);
        load_ws(idB, 0, w0);                           // first chunk of the next pair
        add(e0 + KB, stA, KB, w1);
        idA = idB;                                     // landed at the wait above
        stA = stB;
    }
}

}  // namespace
