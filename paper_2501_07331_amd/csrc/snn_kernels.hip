// HIP kernels of libsnn for gfx950 (CDNA4, wave64).
//
// Decomposition of one EventProp training step (Table 1):
//
//  input_scan       the input projection's delayed currents do not depend on
//                   the network state: for every (sample, block of layer-1
//                   posts) a workgroup walks the sample's input spikes in
//                   order through a delay ring in LDS and writes the arrivals
//                   of every step to A_in[b][n][j].  Time-parallel over
//                   samples and post blocks.
//  forward_core     one workgroup per sample runs the LIF layers over T steps:
//                   free dynamics, threshold, wave-ballot spike masks (one
//                   barrier per step), spike records, delayed scatter of the
//                   LIF spikes into per-projection rings, arrivals.
//  readout_forward  the LI readout layer is fed by spikes but feeds nothing
//                   back: it runs after the core from the spike records.
//  loss             softmax cross-entropy on the readout, its adjoint source.
//  readout_adjoint  the readout adjoints (sources only, no jumps) over T, and
//                   for every spike of the layer feeding the readout the
//                   readout part of its lambda_V jump sum.
//  backward_core    one workgroup per sample runs the LIF adjoints in reverse
//                   time: free adjoint dynamics, delayed postsynaptic sums at
//                   the spikes, lambda_V jumps; writes the adjoint trajectory.
//  group            spikes of every sample grouped by presynaptic neuron.
//  gradients        one workgroup per (projection, post neuron j): for every
//                   presynaptic neuron i, sums lambda_I and w (lambda_I -
//                   lambda_V) of post j at the delayed arrivals of i's spikes:
//                   fp32 within a sample in spike order, fp64 over the batch
//                   in sample order; no atomics, deterministic.
//
// Rings are [slot][neuron] with one owning lane per column: scatter and
// gather need no atomics and no barriers, every cell sums its contributions
// in emission order, and a wave's LDS accesses hit 64 consecutive words of
// one row, conflict-free.
#include "snn_internal.h"

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

__device__ __forceinline__ double wave_sum(double x) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off, 64);
    return x;
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

// ------------------------------------------------------------------ small kernels

__global__ void reset_status_kernel(DevStatus* st) {
    if (threadIdx.x == 0) {
        st->bad_input = 0;
        st->overflow = 0;
        st->clamped = 0;
        st->degenerate = 0;
        for (int l = 0; l < SNN_MAX_LAYERS; ++l) st->layer_spikes[l] = 0;
    }
}

// One workgroup per sample: offsets, label, ranges, strict (step, neuron) order.
__global__ void validate_kernel(const int* off, const int* step, const int* neuron, int nnz, int B,
                                int T, int n_in, const int* labels, int C, DevStatus* st) {
    const int b = blockIdx.x;
    const int lo = off[b], hi = off[b + 1];
    bool bad = false;
    if (b == 0 && lo != 0) bad = true;
    if (b == B - 1 && hi != nnz) bad = true;
    if (lo < 0 || hi < lo || hi > nnz) bad = true;
    const int y = labels[b];
    if (y < 0 || y >= C) bad = true;
    if (!bad) {
        for (int e = lo + (int)threadIdx.x; e < hi; e += blockDim.x) {
            const int s = step[e], i = neuron[e];
            if (s < 0 || s >= T || i < 0 || i >= n_in) bad = true;
            if (e > lo) {
                const long long k0 = (long long)step[e - 1] * n_in + neuron[e - 1];
                const long long k1 = (long long)s * n_in + i;
                if (k1 <= k0) bad = true;
            }
        }
    }
    if (bad) atomicOr(&st->bad_input, 1);
}

// idx[b][n] = first input event of sample b with step >= n, n = 0 .. T.
__global__ void step_index_kernel(const int* off, const int* step, int B, int T, int* idx,
                                  const DevStatus* st) {
    if (st->bad_input) return;
    const long long g = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (g >= (long long)B * (T + 1)) return;
    const int b = (int)(g / (T + 1)), n = (int)(g % (T + 1));
    int lo = off[b], hi = off[b + 1];
    while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (step[mid] < n) lo = mid + 1; else hi = mid;
    }
    idx[g] = lo;
}

struct RoundArgs {
    const float* D[SNN_MAXP];
    long long woff[SNN_MAXP + 1];
    int P, max_delay;
};

// Delays are integer multiples of the time step: rint (half to even), clamp.
__global__ void round_delays_kernel(RoundArgs a, uint8_t* slot, DevStatus* st) {
    const long long g = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    bool clamped = false;
    if (g < a.woff[a.P]) {
        int p = 0;
        while (g >= a.woff[p + 1]) ++p;
        const float r = rintf(a.D[p][g - a.woff[p]]);
        int s;
        if (!(r >= 0.0f)) { s = 0; clamped = true; }            // negative or NaN
        else if (r > (float)a.max_delay) { s = a.max_delay; clamped = true; }
        else s = (int)r;
        slot[g] = (uint8_t)s;
    }
    const unsigned long long m = __ballot(clamped);
    if ((threadIdx.x & 63) == 0 && m) atomicAdd(&st->clamped, (unsigned long long)__popcll(m));
}

// ------------------------------------------------------------------ input scan

// Workgroup (sample b, posts [j0, j0 + nb) of layer 1); lane owns post j.
__global__ void __launch_bounds__(256) input_scan_kernel(InScanArgs a) {
    const Topo& t = a.t;
    if (a.st->bad_input) return;
    const int n1 = t.n[1], S = t.S, T = t.T, nb = a.nb;
    const int nblk = (n1 + nb - 1) / nb;
    const int b = blockIdx.x / nblk, tid = threadIdx.x;
    const int j = (blockIdx.x % nblk) * nb + tid;
    const bool live = tid < nb && j < n1;
    lds_f32* col = (lds_f32*)smem + tid;                      // ring [S][nb]
    if (live)
        for (int s = 0; s < S; ++s) col[s * nb] = 0.0f;
    const int* idx = a.in_idx + (size_t)b * (T + 1);
    global_f32* out = (global_f32*)(a.A_in + (size_t)b * T * n1 + (live ? j : 0));
    int e_lo = uniform32(idx[0]);
    int n_mod = 0;
    for (int n = 0; n < T; ++n) {
        const int e_hi = uniform32(idx[n + 1]);
        for (int e0 = e_lo; e0 < e_hi; e0 += KB) {
            int ids[KB], row[KB];
            float w[KB];
            list_chunk(a.in_neuron, e0, e_hi, ids);
            if (live) {
                chunk_rows(a.W0, a.slot0, n1, j, n, n_mod, S, T, ids, row, w);
                column_add(col, nb, row, w);
            }
        }
        if (live) {
            out[(size_t)n * n1] = col[n_mod * nb];
            col[n_mod * nb] = 0.0f;
        }
        e_lo = e_hi;
        n_mod = (n_mod + 1 == S) ? 0 : n_mod + 1;
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

__device__ __forceinline__ bool bits_chunk(BitIter& it, int (&ids)[KB]) {
    bool any = false;
#pragma unroll
    for (int k = 0; k < KB; ++k) {
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

template <int MAXT>
__global__ void __launch_bounds__(MAXT) forward_core_kernel(CoreFwdArgs a) {
    const Topo& t = a.t;
    if (a.st->bad_input) return;
    const int b = blockIdx.x, tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6, nwaves = blockDim.x >> 6;
    float* lds = reinterpret_cast<float*>(smem);
    unsigned long long* masks = reinterpret_cast<unsigned long long*>(smem + a.mask_off);
    const int S = t.S, T = t.T, L = t.L;

    // zero the ring columns this lane owns
    for (int p = 0; p < t.P; ++p) {
        const int q = t.post[p], nq = t.n[q];
        if (t.pre[p] == 0 || t.kind[q] != SNN_LIF || tid >= nq) continue;
        if (t.fring[p] >= 0) {
            lds_f32* c = (lds_f32*)(lds + t.fring[p]) + tid;
            for (int s = 0; s < S; ++s) c[s * nq] = 0.0f;
        } else {
            global_f32* c = (global_f32*)(a.ring[p] + (size_t)b * S * nq) + tid;
            for (int s = 0; s < S; ++s) c[s * nq] = 0.0f;
        }
    }

    float V[SNN_MAX_LAYERS], I[SNN_MAX_LAYERS];
    bool spk[SNN_MAX_LAYERS];
    int cnt[SNN_MAX_LAYERS];
#pragma unroll
    for (int l = 0; l < SNN_MAX_LAYERS; ++l) {
        V[l] = 0.0f;
        I[l] = 0.0f;
        spk[l] = false;
        cnt[l] = 0;
    }
    const int n1 = t.n[1];
    const global_f32* ain = (const global_f32*)(a.A_in + (size_t)b * T * n1) + tid;
    float ain_next = (tid < n1) ? ain[0] : 0.0f;
    int n_mod = 0;

    for (int n = 0; n < T; ++n) {
        const int par = n & 1;
        const float ain_n = ain_next;
        if (tid < n1 && n + 1 < T) ain_next = ain[(size_t)(n + 1) * n1];
        // ---- free dynamics over one step, threshold, reset
#pragma unroll
        for (int l = 1; l < SNN_MAX_LAYERS; ++l) {
            if (l >= L || t.kind[l] != SNN_LIF) break;
            bool s_ = false;
            if (tid < t.n[l]) {
                const float gi = __fmul_rn(t.gamma, I[l]);
                const float Vm = __fmaf_rn(t.alpha, V[l], gi);
                I[l] = __fmul_rn(t.beta, I[l]);
                s_ = Vm >= t.theta;
                V[l] = s_ ? 0.0f : Vm;
            }
            spk[l] = s_;
            const unsigned long long m = __ballot(s_);
            if (lane == 0) masks[((size_t)par * t.n_lif + t.lif[l]) * nwaves + wave] = m;
        }
        __syncthreads();

        // ---- spike records (ascending neuron order: waves ascending, lanes ascending)
#pragma unroll
        for (int l = 1; l < SNN_MAX_LAYERS; ++l) {
            if (l >= L || t.kind[l] != SNN_LIF) break;
            const int li = t.lif[l];
            const unsigned long long* mk = masks + ((size_t)par * t.n_lif + li) * nwaves;
            int before = 0, total = 0;
            for (int w = 0; w < nwaves; ++w) {
                const int c = __popcll(uniform64(mk[w]));
                before += (w < wave) ? c : 0;
                total += c;
            }
            // internal record indices never pass the capacity (the caller's
            // count stays exact)
            if (tid == 0) a.rec_idx[((size_t)li * t.B + b) * (T + 1) + n] = min(cnt[l], t.cap);
            if (spk[l]) {
                const int pos = cnt[l] + before + lanes_below(mk[wave]);
                if (pos < t.cap) {
                    const size_t r = ((size_t)li * t.B + b) * t.cap + pos;
                    a.rec_n[r] = tid;
                    a.rec_s[r] = n;
                    a.rec_I[r] = I[l];
                    const size_t o = (size_t)b * t.cap + pos;
                    a.out_step[l][o] = n;
                    a.out_neuron[l][o] = tid;
                }
            }
            if (tid == 0 && cnt[l] + total > t.cap) a.st->overflow = 1;
            cnt[l] += total;
        }

        // ---- delayed scatter of the LIF spikes into the LIF-post rings
        for (int p = 0; p < t.P; ++p) {
            const int pa = t.pre[p], q = t.post[p], nq = t.n[q];
            if (pa == 0 || t.kind[q] != SNN_LIF || tid >= nq) continue;
            const float* Wp = a.W[p];
            const uint8_t* Sp = a.slot + t.woff[p];
            BitIter it = bits_begin(masks + ((size_t)par * t.n_lif + t.lif[pa]) * nwaves, nwaves);
            int ids[KB], row[KB];
            float w[KB];
            while (bits_chunk(it, ids)) {
                chunk_rows(Wp, Sp, nq, tid, n, n_mod, S, T, ids, row, w);
                if (t.fring[p] >= 0)
                    column_add((lds_f32*)(lds + t.fring[p]) + tid, nq, row, w);
                else
                    column_add((global_f32*)(a.ring[p] + (size_t)b * S * nq) + tid, nq, row, w);
            }
        }

        // ---- arrivals: per projection into the layer, in projection order
        for (int p = 0; p < t.P; ++p) {
            const int q = t.post[p], nq = t.n[q];
            if (t.kind[q] != SNN_LIF || tid >= nq) continue;
            float add;
            if (t.pre[p] == 0) {
                add = ain_n;
            } else if (t.fring[p] >= 0) {
                lds_f32* c = (lds_f32*)(lds + t.fring[p]) + n_mod * nq + tid;
                add = *c;
                *c = 0.0f;
            } else {
                global_f32* c = (global_f32*)(a.ring[p] + ((size_t)b * S + n_mod) * nq) + tid;
                add = *c;
                *c = 0.0f;
            }
#pragma unroll
            for (int l = 1; l < SNN_MAX_LAYERS; ++l)
                if (l == q) I[l] = __fadd_rn(I[l], add);
        }
        n_mod = (n_mod + 1 == S) ? 0 : n_mod + 1;
    }

    // ---- epilogue
    int soff = 0, nstate = 0;
    for (int l = 1; l < L; ++l) nstate += t.n[l];
#pragma unroll
    for (int l = 1; l < SNN_MAX_LAYERS; ++l) {
        if (l >= L || t.kind[l] != SNN_LIF) break;
        if (tid < t.n[l]) {
            a.Vf[(size_t)b * nstate + soff + tid] = V[l];
            a.If[(size_t)b * nstate + soff + tid] = I[l];
        }
        soff += t.n[l];
        if (tid == 0) {
            const int li = t.lif[l];
            a.rec_idx[((size_t)li * t.B + b) * (T + 1) + T] = min(cnt[l], t.cap);
            a.rec_cnt[(size_t)li * t.B + b] = min(cnt[l], t.cap);
            a.out_count[l][b] = cnt[l];
            atomicAdd(&a.st->layer_spikes[li], (unsigned long long)cnt[l]);
        }
    }
}

// ------------------------------------------------------------------ readout

// Readout arrivals of sample b into the column of output k: table cell m at
// col[m * C] for every step m (an arrival table, not a ring: the spikes are
// all known).  Spikes in record (emission) order.
template <typename Ptr>
__device__ __forceinline__ void readout_table(const ReadoutArgs& a, int b, int k, Ptr col) {
    const Topo& t = a.t;
    const int C = t.n[t.out_l], T = t.T;
    const int pa = t.pre[t.out_p];
    const size_t base = ((size_t)t.lif[pa] * t.B + b) * t.cap;
    const int cnt = uniform32(a.rec_idx[((size_t)t.lif[pa] * t.B + b) * (T + 1) + T]);
    for (int k0 = 0; k0 < cnt; k0 += KB) {
        int ids[KB], steps[KB], row[KB];
        float w[KB];
        list_chunk(a.rec_n + base, k0, cnt, ids);
        list_chunk(a.rec_s + base, k0, cnt, steps);
        if (k < C) {
#pragma unroll
            for (int q = 0; q < KB; ++q) {
                row[q] = -1;
                w[q] = 0.0f;
                if (ids[q] >= 0) {
                    const size_t kk = (size_t)ids[q] * C + k;
                    const int m = steps[q] + a.slot[t.woff[t.out_p] + kk];
                    w[q] = a.W[kk];
                    if (m <= T - 1) row[q] = m;
                }
            }
            column_add(col, C, row, w);
        }
    }
}

// One workgroup per sample, lane k owns output neuron k.  table_lds >= 0:
// the arrival table [T][C] lives in LDS; else in the global ring buffer
// (sized [B][T][C] by the host for this case).
__global__ void __launch_bounds__(1024) readout_forward_kernel(ReadoutArgs a) {
    const Topo& t = a.t;
    if (a.st->bad_input) return;
    const int b = blockIdx.x, k = threadIdx.x;
    const int C = t.n[t.out_l], T = t.T;
    const int pa = t.pre[t.out_p];
    float* lds = reinterpret_cast<float*>(smem);
    const bool in_lds = a.table_lds >= 0;
    lds_f32* lcol = (lds_f32*)(lds + (in_lds ? a.table_lds : 0)) + k;
    global_f32* gcol = in_lds ? nullptr : (global_f32*)(a.table + (size_t)b * T * C) + k;
    if (pa != 0) {
        if (k < C) {
            for (int m = 0; m < T; ++m) {
                if (in_lds) lcol[m * C] = 0.0f; else gcol[m * C] = 0.0f;
            }
        }
        if (in_lds) readout_table(a, b, k, lcol); else readout_table(a, b, k, gcol);
    }
    if (k >= C) return;
    const global_f32* ain = (const global_f32*)(a.A_in + (size_t)b * T * C) + k;
    float V = 0.0f, I = 0.0f, acc = 0.0f, best = 0.0f;
    int nst = 0;
    for (int n = 0; n < T; ++n) {
        const float gi = __fmul_rn(t.gamma, I);
        const float Vm = __fmaf_rn(t.alpha, V, gi);
        I = __fmul_rn(t.beta, I);
        V = Vm;
        if (t.loss == SNN_LOSS_CE_SUM) {
            acc = __fadd_rn(acc, Vm);
        } else if (n == 0 || Vm > best) {
            best = Vm;
            nst = n;
        }
        const float add = (pa == 0) ? ain[(size_t)n * C] : (in_lds ? lcol[n * C] : gcol[n * C]);
        I = __fadd_rn(I, add);
    }
    a.z[(size_t)b * C + k] = (t.loss == SNN_LOSS_CE_SUM) ? __fmul_rn(t.rscale, acc) : best;
    a.nstar[(size_t)b * C + k] = (t.loss == SNN_LOSS_CE_SUM) ? -1 : nst;
    int nstate = 0;
    for (int l = 1; l < t.L; ++l) nstate += t.n[l];
    a.Vf[(size_t)b * nstate + (nstate - C) + k] = V;
    a.If[(size_t)b * nstate + (nstate - C) + k] = I;
}

// ------------------------------------------------------------------ loss

// Softmax cross-entropy on z in fp64; loss_out[b], loss_out[B] = mean; the
// per-step loss source on the readout adjoint src = s g / tau_m (sum) or
// g / tau_m (max), g = (softmax - onehot) / B rounded to fp32 first.
__global__ void loss_kernel(const float* z, const int* labels, int B, int C, int loss, float rscale,
                            float tau_m, float* loss_out, float* src, const DevStatus* st) {
    __shared__ double part[256];
    if (st->bad_input) return;
    double tot = 0.0;
    for (int b = threadIdx.x; b < B; b += blockDim.x) {
        const float* zb = z + (size_t)b * C;
        double mx = zb[0];
        for (int k = 1; k < C; ++k) mx = fmax(mx, (double)zb[k]);
        double se = 0.0;
        for (int k = 0; k < C; ++k) se += exp((double)zb[k] - mx);
        const double lse = mx + log(se);
        const int y = labels[b];
        const double ce = lse - (double)zb[y];
        loss_out[b] = (float)ce;
        tot += ce;
        for (int k = 0; k < C; ++k) {
            const double p = exp((double)zb[k] - lse);
            const float g = (float)((p - (k == y ? 1.0 : 0.0)) / (double)B);
            const double sk = (loss == SNN_LOSS_CE_SUM) ? (double)rscale * (double)g / (double)tau_m
                                                        : (double)g / (double)tau_m;
            src[(size_t)b * C + k] = (float)sk;
        }
    }
    part[threadIdx.x] = tot;
    __syncthreads();
    for (int w = blockDim.x / 2; w > 0; w >>= 1) {
        if ((int)threadIdx.x < w) part[threadIdx.x] += part[threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x == 0) loss_out[B] = (float)(part[0] / (double)B);
}

// ------------------------------------------------------------------ readout adjoint

// One workgroup per sample, lane k owns output neuron k.  The readout
// adjoints see only their loss source: lambda_I, lambda_V over reverse time
// (the "+" values before the step's source are the trajectory), then the
// readout part of the jump sum of every spike (n, i) of the feeding LIF
// layer: A2 = sum_k w_ik (lambda_V - lambda_I)_k at n + slot_ik (fp64 sum).
__global__ void __launch_bounds__(1024) readout_adjoint_kernel(ReadoutArgs a) {
    const Topo& t = a.t;
    const int b = blockIdx.x, k = threadIdx.x, lane = k & 63;
    const int C = t.n[t.out_l], T = t.T;
    const int pa = t.pre[t.out_p];
    const int nwaves = blockDim.x >> 6;
    float* lds = reinterpret_cast<float*>(smem);
    const bool in_lds = a.table_lds >= 0;
    lds_f32* tab = (lds_f32*)(lds + (in_lds ? a.table_lds : 0));
    global_f32* tu = (global_f32*)(a.tu + ((size_t)b * C + k) * T);
    global_f32* td = (global_f32*)(a.td + ((size_t)b * C + k) * T);
    if (k < C) {
        const float srcv = a.src[(size_t)b * C + k];
        const int nst = a.nstar[(size_t)b * C + k];
        float lv = 0.0f, lI = 0.0f;
        for (int n = T - 1; n >= 0; --n) {
            if (n <= T - 2) {
                const float v = lv;
                lI = __fadd_rn(__fmul_rn(t.beta, lI), __fmul_rn(t.cc, v));
                lv = __fmul_rn(t.alpha, v);
            }
            const float d = __fsub_rn(lI, lv);
            tu[n] = lI;
            td[n] = d;
            if (in_lds) tab[n * C + k] = d;
            if (t.loss == SNN_LOSS_CE_SUM || nst == n) lv = __fsub_rn(lv, srcv);
        }
    }
    if (pa == 0) return;
    __syncthreads();
    double* red = reinterpret_cast<double*>(smem + a.red_off);    // [KB] fp64 partial sums
    const size_t base = ((size_t)t.lif[pa] * t.B + b) * t.cap;
    double* A2 = a.A2 + (size_t)b * t.cap;
    const int cnt = uniform32(a.rec_idx[((size_t)t.lif[pa] * t.B + b) * (T + 1) + T]);
    for (int k0 = 0; k0 < cnt; k0 += KB) {
        int ids[KB], steps[KB];
        list_chunk(a.rec_n + base, k0, cnt, ids);
        list_chunk(a.rec_s + base, k0, cnt, steps);
        double part[KB];
#pragma unroll
        for (int q = 0; q < KB; ++q) {
            part[q] = 0.0;
            if (ids[q] >= 0 && k < C) {
                const size_t kk = (size_t)ids[q] * C + k;
                const int m = steps[q] + a.slot[t.woff[t.out_p] + kk];
                if (m <= T - 1) {
                    const float d = in_lds ? (float)tab[m * C + k] : (float)td[m];
                    part[q] = -(double)__fmul_rn(a.W[kk], d);
                }
            }
        }
        if (nwaves == 1) {
#pragma unroll
            for (int q = 0; q < KB; ++q) {
                const double s = wave_sum(part[q]);
                if (ids[q] >= 0 && lane == 0) A2[k0 + q] = s;
            }
        } else {
            if (k < KB) red[k] = 0.0;
            __syncthreads();
#pragma unroll
            for (int q = 0; q < KB; ++q) {
                const double s = wave_sum(part[q]);
                if (ids[q] >= 0 && lane == 0) lds_add_f64(&red[q], s);
            }
            __syncthreads();
            if (k < KB) {
#pragma unroll
                for (int q = 0; q < KB; ++q)
                    if (q == k && ids[q] >= 0) A2[k0 + q] = red[q];
            }
            __syncthreads();
        }
    }
}

// ------------------------------------------------------------------ backward core

template <int MAXT>
__global__ void __launch_bounds__(MAXT) backward_core_kernel(CoreBwdArgs a) {
    const Topo& t = a.t;
    const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63;
    const int S = t.S, T = t.T, L = t.L;
    float* lds = reinterpret_cast<float*>(smem);
    double* accL = reinterpret_cast<double*>(smem + a.acc_off);   // [2][lif_total]
    for (int i = tid; i < 2 * t.lif_total; i += blockDim.x) accL[i] = 0.0;
    __syncthreads();
    const int feed = t.pre[t.out_p];          // LIF layer feeding the readout (0: none)

    float lv[SNN_MAX_LAYERS], lI[SNN_MAX_LAYERS];
#pragma unroll
    for (int l = 0; l < SNN_MAX_LAYERS; ++l) { lv[l] = 0.0f; lI[l] = 0.0f; }
    unsigned long long deg = 0;
    int n_mod = (T - 1) % S;

    for (int n = T - 1; n >= 0; --n) {
        const int par = n & 1;
        // ---- adjoint free dynamics, trajectory, ring
#pragma unroll
        for (int l = 1; l < SNN_MAX_LAYERS; ++l) {
            if (l >= L || t.kind[l] != SNN_LIF) break;
            const int nl = t.n[l];
            if (tid >= nl) continue;
            if (n <= T - 2) {
                const float v = lv[l];
                lI[l] = __fadd_rn(__fmul_rn(t.beta, lI[l]), __fmul_rn(t.cc, v));
                lv[l] = __fmul_rn(t.alpha, v);
            }
            const float d = __fsub_rn(lI[l], lv[l]);
            const size_t o = ((size_t)b * t.lif_total + t.lif_off[l] + tid) * T + n;
            a.tu[o] = lI[l];
            a.td[o] = d;
            if (t.bring[l] >= 0) ((lds_f32*)(lds + t.bring[l]))[n_mod * nl + tid] = d;
            else if (a.ring[l]) ((global_f32*)(a.ring[l] + ((size_t)b * S + n_mod) * nl))[tid] = d;
        }
        // ---- postsynaptic sums of the LIF spikes of this step
#pragma unroll
        for (int l = 1; l < SNN_MAX_LAYERS; ++l) {
            if (l >= L || t.kind[l] != SNN_LIF) break;
            const int li = t.lif[l];
            const int* ri = a.rec_idx + ((size_t)li * t.B + b) * (T + 1);
            const int k_lo = uniform32(ri[n]), k_hi = uniform32(ri[n + 1]);
            const int* rn = a.rec_n + ((size_t)li * t.B + b) * t.cap;
            for (int k0 = k_lo; k0 < k_hi; k0 += KB) {
                int ids[KB];
                list_chunk(rn, k0, k_hi, ids);
                double part[KB];
#pragma unroll
                for (int k = 0; k < KB; ++k) part[k] = 0.0;
                for (int p = 0; p < t.P; ++p) {
                    const int q = t.post[p], nq = t.n[q];
                    if (t.pre[p] != l || t.kind[q] != SNN_LIF || tid >= nq) continue;
                    int row[KB];
                    float w[KB];
                    chunk_rows(a.W[p], a.slot + t.woff[p], nq, tid, n, n_mod, S, T, ids, row, w);
#pragma unroll
                    for (int k = 0; k < KB; ++k) {
                        if (row[k] < 0) continue;
                        const float d = (t.bring[q] >= 0)
                            ? (float)((lds_f32*)(lds + t.bring[q]))[row[k] * nq + tid]
                            : (float)((global_f32*)(a.ring[q] + ((size_t)b * S + row[k]) * nq))[tid];
                        part[k] -= (double)__fmul_rn(w[k], d);
                    }
                }
#pragma unroll
                for (int k = 0; k < KB; ++k) {
                    if (ids[k] < 0) continue;
                    const double sum = wave_sum(part[k]);
                    if (lane == 0 && sum != 0.0)
                        lds_add_f64(&accL[par * t.lif_total + t.lif_off[l] + ids[k]], sum);
                }
            }
        }
        __syncthreads();
        // ---- lambda_V jumps at the spikes of this step
#pragma unroll
        for (int l = 1; l < SNN_MAX_LAYERS; ++l) {
            if (l >= L || t.kind[l] != SNN_LIF) break;
            const int li = t.lif[l];
            const int* ri = a.rec_idx + ((size_t)li * t.B + b) * (T + 1);
            const int k_lo = uniform32(ri[n]), k_hi = uniform32(ri[n + 1]);
            const size_t base = ((size_t)li * t.B + b) * t.cap;
            for (int kr = k_lo; kr < k_hi; ++kr) {
                if (a.rec_n[base + kr] != tid) continue;
                double* ap = &accL[par * t.lif_total + t.lif_off[l] + tid];
                double A = *ap;
                *ap = 0.0;
                if (l == feed) A += a.A2[(size_t)b * t.cap + kr];
                const float den = __fsub_rn(a.rec_I[base + kr], t.theta);
                if (den > 0.0f) {
                    const float D = (float)(((double)t.theta * (double)lv[l] + A) / (double)den);
                    lv[l] = __fadd_rn(lv[l], D);
                } else {
                    ++deg;
                }
            }
        }
        n_mod = (n_mod == 0) ? S - 1 : n_mod - 1;
    }
    if (deg) atomicAdd(&a.st->degenerate, deg);
}

// ------------------------------------------------------------------ grouping

// One workgroup per sample: counting sort of the sample's spikes by
// presynaptic neuron (LDS histogram), then each neuron's steps sorted.
__global__ void __launch_bounds__(1024) group_kernel(GroupArgs a) {
    if (a.st->bad_input) return;
    const int b = blockIdx.x, tid = threadIdx.x, nt = blockDim.x;
    const int start = a.cnt ? b * a.off_stride : a.off[b];
    const int end = a.cnt ? start + a.cnt[b] : a.end[b + 1];
    int* h = reinterpret_cast<int*>(smem);        // [n + 1] counts, then cursors
    int* part = h + a.n + 1;                      // [nt] block scan
    for (int i = tid; i <= a.n; i += nt) h[i] = 0;
    __syncthreads();
    for (int e = start + tid; e < end; e += nt) atomicAdd(&h[a.neuron[e]], 1);
    __syncthreads();
    // exclusive scan of h[0 .. n): thread tid scans a contiguous segment
    const int seg = (a.n + nt - 1) / nt;
    const int i0 = min(tid * seg, a.n), i1 = min(i0 + seg, a.n);
    int s = 0;
    for (int i = i0; i < i1; ++i) s += h[i];
    part[tid] = s;
    __syncthreads();
    if (tid == 0) {
        int run = 0;
        for (int w = 0; w < nt; ++w) {
            const int v = part[w];
            part[w] = run;
            run += v;
        }
    }
    __syncthreads();
    int run = part[tid];
    int* goff = a.g_off + (size_t)b * (a.n + 1);
    for (int i = i0; i < i1; ++i) {
        const int v = h[i];
        h[i] = run;
        goff[i] = start + run;
        run += v;
    }
    if (tid == 0) goff[a.n] = end;
    __syncthreads();
    for (int e = start + tid; e < end; e += nt) {
        const int pos = atomicAdd(&h[a.neuron[e]], 1);
        a.g_step[start + pos] = a.step[e];
    }
    __syncthreads();
    for (int i = tid; i < a.n; i += nt) {
        const int lo = goff[i], hi = goff[i + 1];
        for (int x = lo + 1; x < hi; ++x) {
            const int v = a.g_step[x];
            int y = x - 1;
            while (y >= lo && a.g_step[y] > v) {
                a.g_step[y + 1] = a.g_step[y];
                --y;
            }
            a.g_step[y + 1] = v;
        }
    }
}

// ------------------------------------------------------------------ gradients

// Workgroup = (projection p, post neuron j); lane = presynaptic neuron i
// (i = i0 + tid for passes i0 over the pre layer).  Per sample: the post
// adjoint trajectory is staged in LDS, then every lane sums over its spikes
// (ascending steps) lambda_I and w (lambda_I - lambda_V) at the arrival steps
// in fp32, and adds the per-sample sums to fp64 totals.
__global__ void __launch_bounds__(1024) gradients_kernel(GradArgs a) {
    const Topo& t = a.t;
    int p = 0;
    while ((int)blockIdx.x >= a.blk[p + 1]) ++p;
    const int j = blockIdx.x - a.blk[p];
    const int pa = t.pre[p], q = t.post[p];
    const int npre = t.n[pa], nq = t.n[q], T = t.T, tid = threadIdx.x;
    const bool lif_post = t.kind[q] == SNN_LIF;
    lds_f32* U = (lds_f32*)smem;
    lds_f32* Dd = U + T;
    const int* goff = a.g_off[pa];
    const int* gstep = a.g_step[pa];
    for (int i0 = 0; i0 < npre; i0 += blockDim.x) {
        const int i = i0 + tid;
        const bool live = i < npre;
        float w = 0.0f;
        int s = 0;
        if (live) {
            w = a.W[p][(size_t)i * nq + j];
            s = a.slot[t.woff[p] + (size_t)i * nq + j];
        }
        double su = 0.0, sd = 0.0;
        for (int b = 0; b < t.B; ++b) {
            const size_t o = lif_post ? ((size_t)b * t.lif_total + t.lif_off[q] + j) * T
                                      : ((size_t)b * nq + j) * T;
            const float* tu = lif_post ? a.tu_lif : a.tu_out;
            const float* td = lif_post ? a.td_lif : a.td_out;
            __syncthreads();
            for (int m = tid; m < T; m += blockDim.x) {
                U[m] = tu[o + m];
                Dd[m] = td[o + m];
            }
            __syncthreads();
            if (!live) continue;
            const int* g = goff + (size_t)b * (npre + 1) + i;
            const int lo = g[0], hi = g[1];
            float pu = 0.0f, pd = 0.0f;
            for (int x = lo; x < hi; ++x) {
                const int m = gstep[x] + s;
                if (m > T - 1) break;                  // steps ascend
                pu = __fadd_rn(pu, U[m]);
                pd = __fadd_rn(pd, __fmul_rn(w, Dd[m]));
            }
            su += (double)pu;
            sd += (double)pd;
        }
        if (live) {
            a.dW[p][(size_t)i * nq + j] = (float)(-(double)t.tau_s * su);
            a.dD[p][(size_t)i * nq + j] = (float)(-(double)t.dt * sd);
        }
    }
}

__global__ void copy_state_kernel(const float* src, int stride, int off, int n, int B, float* dst) {
    const long long g = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (g >= (long long)B * n) return;
    const long long b = g / n, j = g % n;
    dst[g] = src[b * stride + off + j];
}

}  // namespace

// ------------------------------------------------------------------ launchers

hipError_t launch_reset_status(DevStatus* st, hipStream_t s) {
    hipLaunchKernelGGL(reset_status_kernel, dim3(1), dim3(64), 0, s, st);
    return hipGetLastError();
}

hipError_t launch_validate(const int* off, const int* step, const int* neuron, int nnz, int B, int T,
                           int n_in, const int* labels, int C, DevStatus* st, hipStream_t s) {
    hipLaunchKernelGGL(validate_kernel, dim3(B), dim3(256), 0, s, off, step, neuron, nnz, B, T, n_in,
                       labels, C, st);
    return hipGetLastError();
}

hipError_t launch_step_index(const int* off, const int* step, int B, int T, int* idx,
                             const DevStatus* st, hipStream_t s) {
    const long long n = (long long)B * (T + 1);
    hipLaunchKernelGGL(step_index_kernel, dim3(grid_for(n, 256)), dim3(256), 0, s, off, step, B, T,
                       idx, st);
    return hipGetLastError();
}

hipError_t launch_round_delays(const float* const* D, const long long* woff, const long long* cnt,
                               int P, int max_delay, uint8_t* slot, DevStatus* st, hipStream_t s) {
    RoundArgs a{};
    for (int p = 0; p < P; ++p) {
        a.D[p] = D[p];
        a.woff[p] = woff[p];
    }
    a.woff[P] = woff[P - 1] + cnt[P - 1];
    a.P = P;
    a.max_delay = max_delay;
    hipLaunchKernelGGL(round_delays_kernel, dim3(grid_for(a.woff[P], 256)), dim3(256), 0, s, a, slot,
                       st);
    return hipGetLastError();
}

hipError_t launch_input_scan(const InScanArgs& a, size_t lds, hipStream_t s) {
    const int nblk = (a.t.n[1] + a.nb - 1) / a.nb;
    const int threads = ((a.nb + 63) / 64) * 64;
    hipLaunchKernelGGL(input_scan_kernel, dim3(a.t.B * nblk), dim3(threads), lds, s, a);
    return hipGetLastError();
}

// Workgroups of up to 256 threads get the 256-thread instantiation (one wave
// per SIMD, up to 512 registers per lane); wider networks the 1024-thread one.
hipError_t launch_forward_core(const CoreFwdArgs& a, int threads, size_t lds, hipStream_t s) {
    if (threads <= 256)
        hipLaunchKernelGGL(forward_core_kernel<256>, dim3(a.t.B), dim3(threads), lds, s, a);
    else
        hipLaunchKernelGGL(forward_core_kernel<1024>, dim3(a.t.B), dim3(threads), lds, s, a);
    return hipGetLastError();
}

hipError_t launch_readout_forward(const ReadoutArgs& a, int threads, size_t lds, hipStream_t s) {
    hipLaunchKernelGGL(readout_forward_kernel, dim3(a.t.B), dim3(threads), lds, s, a);
    return hipGetLastError();
}

hipError_t launch_loss(const float* z, const int* labels, int B, int C, int loss, float rscale,
                       float tau_m, float* loss_out, float* src, const DevStatus* st, hipStream_t s) {
    hipLaunchKernelGGL(loss_kernel, dim3(1), dim3(256), 0, s, z, labels, B, C, loss, rscale, tau_m,
                       loss_out, src, st);
    return hipGetLastError();
}

hipError_t launch_readout_adjoint(const ReadoutArgs& a, int threads, size_t lds, hipStream_t s) {
    hipLaunchKernelGGL(readout_adjoint_kernel, dim3(a.t.B), dim3(threads), lds, s, a);
    return hipGetLastError();
}

hipError_t launch_backward_core(const CoreBwdArgs& a, int threads, size_t lds, hipStream_t s) {
    if (threads <= 256)
        hipLaunchKernelGGL(backward_core_kernel<256>, dim3(a.t.B), dim3(threads), lds, s, a);
    else
        hipLaunchKernelGGL(backward_core_kernel<1024>, dim3(a.t.B), dim3(threads), lds, s, a);
    return hipGetLastError();
}

hipError_t launch_group(const GroupArgs& a, int B, hipStream_t s) {
    const size_t lds = sizeof(int) * ((size_t)a.n + 1 + 1024);
    hipLaunchKernelGGL(group_kernel, dim3(B), dim3(1024), lds, s, a);
    return hipGetLastError();
}

hipError_t launch_gradients(const GradArgs& a, int blocks, size_t lds, hipStream_t s) {
    int maxpre = 64;
    for (int p = 0; p < a.t.P; ++p) maxpre = maxpre > a.t.n[a.t.pre[p]] ? maxpre : a.t.n[a.t.pre[p]];
    const int threads = maxpre >= 1024 ? 1024 : ((maxpre + 63) / 64) * 64;
    hipLaunchKernelGGL(gradients_kernel, dim3(blocks), dim3(threads), lds, s, a);
    return hipGetLastError();
}

hipError_t launch_copy_state(const float* src, int stride, int off, int n, int B, float* dst,
                             hipStream_t s) {
    hipLaunchKernelGGL(copy_state_kernel, dim3(grid_for((long long)B * n, 256)), dim3(256), 0, s, src,
                       stride, off, n, B, dst);
    return hipGetLastError();
}

hipError_t set_kernel_lds_limits(size_t bytes) {
    const void* fns[] = {(const void*)input_scan_kernel,          (const void*)forward_core_kernel<256>,
                         (const void*)forward_core_kernel<1024>,  (const void*)readout_forward_kernel,
                         (const void*)readout_adjoint_kernel,     (const void*)backward_core_kernel<256>,
                         (const void*)backward_core_kernel<1024>, (const void*)group_kernel,
                         (const void*)gradients_kernel};
    for (const void* f : fns) {
        const hipError_t e =
            hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}
