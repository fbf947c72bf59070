// HIP kernels of libsnn for gfx950 (CDNA4, wave64).
//
// Layout: one workgroup per sample runs all T steps; lane t of the workgroup
// owns neuron t of every non-input layer.  A delay ring R[S][n] (fp32) per
// post layer and sample is indexed [slot][neuron], so every ring column has a
// single owning lane: scatter and gather need no atomics and no barriers, the
// fp32 summation order of every cell is the fixed (emission step, projection,
// presynaptic index) order, and LDS accesses of a wave hit 64 consecutive
// words of one row, conflict-free whatever the delays.  Rings live in LDS
// when they fit (160 KiB per workgroup on gfx950), otherwise in HBM.
//
// Forward (Table 1 forward dynamics): per step, LIF update and threshold,
// wave-ballot spike masks in LDS (one barrier per step), spike records,
// delayed scatter of the input and LIF spikes of the step into the rings,
// arrivals, readout.
//
// Backward (Table 1 backward dynamics, gradient updates), two passes:
//  A: adjoint propagation in reverse time, ring of d = lambda_I - lambda_V,
//     gathers at the delayed arrival times, dD sums (fp64 atomics), the
//     postsynaptic sum of every LIF spike reduced across the workgroup in
//     fp64, and the lambda_V jump; the jump of every spike is stored.
//  B: the same adjoint trajectory replayed with the stored jumps (no
//     cross-lane dependency, no barrier), ring of lambda_I, dW sums.
// Each pass then needs one fp32 ring, which fits in LDS for the 256-neuron
// recurrent layer of the SHD-sized network (151 x 256 x 4 B).
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

// fp64 atomic adds with the address space stated, so the compiler emits
// global_atomic_add_f64 / ds_add_f64 directly (no flat-address dispatch).
typedef __attribute__((address_space(1))) double global_f64;
typedef __attribute__((address_space(3))) double lds_f64;
// Ring cells are reached through pointers typed with their address space, so
// an LDS access and a global access are never folded into one flat access.
typedef __attribute__((address_space(1))) float global_f32;
typedef __attribute__((address_space(3))) float lds_f32;

__device__ __forceinline__ void global_add_f64(double* p, double v) {
    __hip_atomic_fetch_add((global_f64*)p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void lds_add_f64(double* p, double v) {
    __hip_atomic_fetch_add((lds_f64*)p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

__device__ __forceinline__ double wave_sum(double x) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off, 64);
    return x;
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

// ------------------------------------------------------------------ forward

__device__ __forceinline__ void ring_add(const Topo& t, float* lds, float* const* gr, int b, int q,
                                         int row, int nq, int tid, float w) {
    if (t.ring_lds[q] >= 0) {
        lds_f32* c = (lds_f32*)(lds + t.ring_lds[q] + row * nq + tid);
        *c = __fadd_rn(*c, w);
    } else {
        global_f32* c = (global_f32*)(gr[q] + ((size_t)b * t.S + row) * nq + tid);
        *c = __fadd_rn(*c, w);
    }
}

__global__ void __launch_bounds__(1024) forward_kernel(FwdArgs a) {
    const Topo& t = a.t;
    const int b = blockIdx.x, tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6, nwaves = blockDim.x >> 6;
    if (a.st->bad_input) return;
    float* lds = reinterpret_cast<float*>(smem);
    unsigned long long* masks = reinterpret_cast<unsigned long long*>(smem + a.mask_off);
    const int S = t.S, T = t.T, L = t.L;
    const int* idx = a.in_idx + (size_t)b * (T + 1);

    // zero the ring columns this lane owns
    for (int l = 1; l < L; ++l) {
        const int nl = t.n[l];
        if (tid >= nl) continue;
        if (t.ring_lds[l] >= 0) {
            float* r = lds + t.ring_lds[l];
            for (int s = 0; s < S; ++s) r[s * nl + tid] = 0.0f;
        } else {
            float* r = a.ring[l] + (size_t)b * S * nl;
            for (int s = 0; s < S; ++s) r[s * nl + tid] = 0.0f;
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
    float acc = 0.0f, best = 0.0f;
    int nst = 0;
    int e_lo = idx[0];
    int n_mod = 0;

    for (int n = 0; n < T; ++n) {
        const int par = n & 1;
        // ---- free dynamics over one step, threshold, reset, readout
#pragma unroll
        for (int l = 1; l < SNN_MAX_LAYERS; ++l) {
            if (l >= L) break;
            bool s_ = false;
            if (tid < t.n[l]) {
                const float gi = __fmul_rn(t.gamma, I[l]);
                const float Vm = __fmaf_rn(t.alpha, V[l], gi);
                I[l] = __fmul_rn(t.beta, I[l]);
                if (t.kind[l] == SNN_LIF) {
                    s_ = Vm >= t.theta;
                    V[l] = s_ ? 0.0f : Vm;
                } else {
                    V[l] = Vm;
                }
                if (l == L - 1) {
                    if (t.loss == SNN_LOSS_CE_SUM) {
                        acc = __fadd_rn(acc, Vm);
                    } else if (n == 0 || Vm > best) {
                        best = Vm;
                        nst = n;
                    }
                }
            }
            spk[l] = s_;
            if (t.kind[l] == SNN_LIF) {
                const unsigned long long m = __ballot(s_);
                if (lane == 0) masks[((size_t)par * t.n_lif + t.lif[l]) * nwaves + wave] = m;
            }
        }
        __syncthreads();

        // ---- spike records (ascending neuron order: waves ascending, lanes ascending)
#pragma unroll
        for (int l = 1; l < SNN_MAX_LAYERS; ++l) {
            if (l >= L) break;
            if (t.kind[l] != SNN_LIF) continue;
            const int li = t.lif[l];
            const unsigned long long* mk = masks + ((size_t)par * t.n_lif + li) * nwaves;
            int before = 0, total = 0;
            for (int w = 0; w < nwaves; ++w) {
                const int c = __popcll(uniform64(mk[w]));
                before += (w < wave) ? c : 0;
                total += c;
            }
            if (tid == 0) a.rec_idx[((size_t)li * t.B + b) * (T + 1) + n] = cnt[l];
            if (spk[l]) {
                const int pos = cnt[l] + before + lanes_below(mk[wave]);
                if (pos < t.cap) {
                    const size_t r = ((size_t)li * t.B + b) * t.cap + pos;
                    a.rec_n[r] = tid;
                    a.rec_I[r] = I[l];
                    const size_t o = (size_t)b * t.cap + pos;
                    a.out_step[l][o] = n;
                    a.out_neuron[l][o] = tid;
                }
            }
            if (tid == 0 && cnt[l] + total > t.cap) a.st->overflow = 1;
            cnt[l] += total;
        }

        // ---- delayed scatter: projections in order, presynaptic spikes ascending
        const int e_hi = idx[n + 1];
        for (int p = 0; p < t.P; ++p) {
            const int q = t.post[p], pa = t.pre[p], nq = t.n[q];
            if (tid >= nq) continue;
            const float* Wp = a.W[p];
            const uint8_t* Sp = a.slot + t.woff[p];
            if (pa == 0) {
                for (int e = e_lo; e < e_hi; ++e) {
                    const int i = a.in_neuron[e];
                    const size_t k = (size_t)i * nq + tid;
                    const int s = Sp[k];
                    if (n + s <= T - 1) {
                        int row = n_mod + s;
                        if (row >= S) row -= S;
                        ring_add(t, lds, a.ring, b, q, row, nq, tid, Wp[k]);
                    }
                }
            } else {
                const unsigned long long* mk = masks + ((size_t)par * t.n_lif + t.lif[pa]) * nwaves;
                for (int w = 0; w < nwaves; ++w) {
                    unsigned long long m = uniform64(mk[w]);
                    while (m) {
                        const int i = w * 64 + __builtin_ctzll(m);
                        m &= m - 1;
                        const size_t k = (size_t)i * nq + tid;
                        const int s = Sp[k];
                        if (n + s <= T - 1) {
                            int row = n_mod + s;
                            if (row >= S) row -= S;
                            ring_add(t, lds, a.ring, b, q, row, nq, tid, Wp[k]);
                        }
                    }
                }
            }
        }
        e_lo = e_hi;

        // ---- arrivals at this step
#pragma unroll
        for (int l = 1; l < SNN_MAX_LAYERS; ++l) {
            if (l >= L) break;
            const int nl = t.n[l];
            if (tid >= nl) continue;
            if (t.ring_lds[l] >= 0) {
                float* c = lds + t.ring_lds[l] + n_mod * nl + tid;
                I[l] = __fadd_rn(I[l], *c);
                *c = 0.0f;
            } else {
                float* c = a.ring[l] + ((size_t)b * S + n_mod) * nl + tid;
                I[l] = __fadd_rn(I[l], *c);
                *c = 0.0f;
            }
        }
        n_mod = (n_mod + 1 == S) ? 0 : n_mod + 1;
    }

    // ---- epilogue
    const int C = t.n[L - 1];
    if (tid < C) {
        a.z[(size_t)b * C + tid] = (t.loss == SNN_LOSS_CE_SUM) ? __fmul_rn(t.rscale, acc) : best;
        a.nstar[(size_t)b * C + tid] = (t.loss == SNN_LOSS_CE_SUM) ? -1 : nst;
    }
    int soff = 0, nstate = 0;
    for (int l = 1; l < L; ++l) nstate += t.n[l];
#pragma unroll
    for (int l = 1; l < SNN_MAX_LAYERS; ++l) {
        if (l >= L) break;
        if (tid < t.n[l]) {
            a.Vf[(size_t)b * nstate + soff + tid] = V[l];
            a.If[(size_t)b * nstate + soff + tid] = I[l];
        }
        soff += t.n[l];
        if (t.kind[l] == SNN_LIF && tid == 0) {
            const int li = t.lif[l];
            a.rec_idx[((size_t)li * t.B + b) * (T + 1) + T] = cnt[l];
            a.out_count[l][b] = cnt[l];
            atomicAdd(&a.st->layer_spikes[li], (unsigned long long)cnt[l]);
        }
    }
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

__global__ void fill_f64_kernel(double* p, long long n) {
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (long long)gridDim.x * blockDim.x)
        p[i] = 0.0;
}

// ------------------------------------------------------------------ backward

// Ring cell (row, tid) of layer q for sample b: LDS if the layer's ring lives
// there, else the sample's slice of the global ring.
__device__ __forceinline__ float ring_get(const Topo& t, const float* lds, const float* const* gr,
                                          int b, int q, int row, int nq, int tid) {
    if (t.ring_lds[q] >= 0) return *(const lds_f32*)(lds + t.ring_lds[q] + row * nq + tid);
    return *(const global_f32*)(gr[q] + ((size_t)b * t.S + row) * nq + tid);
}

__device__ __forceinline__ void ring_put(const Topo& t, float* lds, float* const* gr, int b, int q,
                                         int row, int nq, int tid, float v) {
    if (t.ring_lds[q] >= 0) *(lds_f32*)(lds + t.ring_lds[q] + row * nq + tid) = v;
    else *(global_f32*)(gr[q] + ((size_t)b * t.S + row) * nq + tid) = v;
}

// Pass A: adjoints with jumps, dD sums, stored jumps.
__global__ void __launch_bounds__(1024) backward_a_kernel(BwdArgs a) {
    const Topo& t = a.t;
    const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63;
    const int S = t.S, T = t.T, L = t.L, C = t.n[L - 1];
    float* lds = reinterpret_cast<float*>(smem);
    double* accL = reinterpret_cast<double*>(smem + a.acc_off);   // [2][lif_total]
    for (int i = tid; i < 2 * t.lif_total; i += blockDim.x) accL[i] = 0.0;
    __syncthreads();

    float lv[SNN_MAX_LAYERS], lI[SNN_MAX_LAYERS];
#pragma unroll
    for (int l = 0; l < SNN_MAX_LAYERS; ++l) { lv[l] = 0.0f; lI[l] = 0.0f; }
    float srcv = 0.0f;
    int nst = -1;
    if (tid < C) {
        srcv = a.src[(size_t)b * C + tid];
        nst = a.nstar[(size_t)b * C + tid];
    }
    const int* idx = a.in_idx + (size_t)b * (T + 1);
    unsigned long long deg = 0;
    int n_mod = (T - 1) % S;

    for (int n = T - 1; n >= 0; --n) {
        const int par = n & 1;
        // ---- adjoint free dynamics, ring write, loss source
#pragma unroll
        for (int l = 1; l < SNN_MAX_LAYERS; ++l) {
            if (l >= L) break;
            const int nl = t.n[l];
            if (tid >= nl) continue;
            if (n <= T - 2) {
                const float v = lv[l];
                lI[l] = __fadd_rn(__fmul_rn(t.beta, lI[l]), __fmul_rn(t.cc, v));
                lv[l] = __fmul_rn(t.alpha, v);
            }
            ring_put(t, lds, a.ring, b, l, n_mod, nl, tid, __fsub_rn(lI[l], lv[l]));
            if (l == L - 1 && (t.loss == SNN_LOSS_CE_SUM || nst == n)) lv[l] = __fsub_rn(lv[l], srcv);
        }
        // ---- gathers of the input spikes of this step
        const int e_lo = uniform32(idx[n]), e_hi = uniform32(idx[n + 1]);
        for (int p = 0; p < t.P; ++p) {
            if (t.pre[p] != 0) continue;
            const int q = t.post[p], nq = t.n[q];
            if (tid >= nq) continue;
            const float* Wp = a.W[p];
            const uint8_t* Sp = a.slot + t.woff[p];
            double* SDp = a.SD + t.woff[p];
            for (int e = e_lo; e < e_hi; ++e) {
                const int i = a.in_neuron[e];
                const size_t k = (size_t)i * nq + tid;
                const int s = Sp[k];
                if (n + s <= T - 1) {
                    int row = n_mod + s;
                    if (row >= S) row -= S;
                    const float wd = __fmul_rn(Wp[k], ring_get(t, lds, a.ring, b, q, row, nq, tid));
                    global_add_f64(SDp + k, (double)wd);
                }
            }
        }
        // ---- gathers of the LIF spikes of this step, postsynaptic sums
#pragma unroll
        for (int l = 1; l < SNN_MAX_LAYERS; ++l) {
            if (l >= L) break;
            if (t.kind[l] != SNN_LIF) continue;
            const int li = t.lif[l];
            const int* ri = a.rec_idx + ((size_t)li * t.B + b) * (T + 1);
            const int k_lo = uniform32(ri[n]), k_hi = uniform32(ri[n + 1]);
            const int* rn = a.rec_n + ((size_t)li * t.B + b) * t.cap;
            for (int kr = k_lo; kr < k_hi; ++kr) {
                const int i = uniform32(rn[kr]);
                double part = 0.0;
                for (int p = 0; p < t.P; ++p) {
                    if (t.pre[p] != l) continue;
                    const int q = t.post[p], nq = t.n[q];
                    if (tid >= nq) continue;
                    const size_t k = (size_t)i * nq + tid;
                    const int s = a.slot[t.woff[p] + k];
                    if (n + s <= T - 1) {
                        int row = n_mod + s;
                        if (row >= S) row -= S;
                        const float wd =
                            __fmul_rn(a.W[p][k], ring_get(t, lds, a.ring, b, q, row, nq, tid));
                        global_add_f64(a.SD + t.woff[p] + k, (double)wd);
                        part -= (double)wd;
                    }
                }
                part = wave_sum(part);
                if (lane == 0 && part != 0.0) lds_add_f64(&accL[par * t.lif_total + t.lif_off[l] + i], part);
            }
        }
        __syncthreads();
        // ---- lambda_V jumps at the spikes of this step
#pragma unroll
        for (int l = 1; l < SNN_MAX_LAYERS; ++l) {
            if (l >= L) break;
            if (t.kind[l] != SNN_LIF) continue;
            const int li = t.lif[l];
            const int* ri = a.rec_idx + ((size_t)li * t.B + b) * (T + 1);
            const int k_lo = uniform32(ri[n]), k_hi = uniform32(ri[n + 1]);
            const size_t base = ((size_t)li * t.B + b) * t.cap;
            for (int kr = k_lo; kr < k_hi; ++kr) {
                if (a.rec_n[base + kr] != tid) continue;
                double* ap = &accL[par * t.lif_total + t.lif_off[l] + tid];
                const double A = *ap;
                *ap = 0.0;
                const float den = __fsub_rn(a.rec_I[base + kr], t.theta);
                float D = 0.0f;
                if (den > 0.0f) {
                    D = (float)(((double)t.theta * (double)lv[l] + A) / (double)den);
                    lv[l] = __fadd_rn(lv[l], D);
                } else {
                    ++deg;
                }
                a.rec_D[base + kr] = D;
            }
        }
        n_mod = (n_mod == 0) ? S - 1 : n_mod - 1;
    }
    if (deg) atomicAdd(&a.st->degenerate, deg);
}

// Pass B: replay of the adjoint trajectory with the stored jumps, dW sums.
// Every lane only touches its own ring column and its own neurons: no barrier.
__global__ void __launch_bounds__(1024) backward_b_kernel(BwdArgs a) {
    const Topo& t = a.t;
    const int b = blockIdx.x, tid = threadIdx.x;
    const int S = t.S, T = t.T, L = t.L, C = t.n[L - 1];
    float* lds = reinterpret_cast<float*>(smem);
    float lv[SNN_MAX_LAYERS], lI[SNN_MAX_LAYERS];
#pragma unroll
    for (int l = 0; l < SNN_MAX_LAYERS; ++l) { lv[l] = 0.0f; lI[l] = 0.0f; }
    float srcv = 0.0f;
    int nst = -1;
    if (tid < C) {
        srcv = a.src[(size_t)b * C + tid];
        nst = a.nstar[(size_t)b * C + tid];
    }
    const int* idx = a.in_idx + (size_t)b * (T + 1);
    int n_mod = (T - 1) % S;

    for (int n = T - 1; n >= 0; --n) {
#pragma unroll
        for (int l = 1; l < SNN_MAX_LAYERS; ++l) {
            if (l >= L) break;
            const int nl = t.n[l];
            if (tid >= nl) continue;
            if (n <= T - 2) {
                const float v = lv[l];
                lI[l] = __fadd_rn(__fmul_rn(t.beta, lI[l]), __fmul_rn(t.cc, v));
                lv[l] = __fmul_rn(t.alpha, v);
            }
            ring_put(t, lds, a.ring, b, l, n_mod, nl, tid, lI[l]);
            if (l == L - 1 && (t.loss == SNN_LOSS_CE_SUM || nst == n)) lv[l] = __fsub_rn(lv[l], srcv);
        }
        const int e_lo = uniform32(idx[n]), e_hi = uniform32(idx[n + 1]);
        for (int p = 0; p < t.P; ++p) {
            if (t.pre[p] != 0) continue;
            const int q = t.post[p], nq = t.n[q];
            if (tid >= nq) continue;
            const uint8_t* Sp = a.slot + t.woff[p];
            double* SUp = a.SU + t.woff[p];
            for (int e = e_lo; e < e_hi; ++e) {
                const int i = a.in_neuron[e];
                const size_t k = (size_t)i * nq + tid;
                const int s = Sp[k];
                if (n + s <= T - 1) {
                    int row = n_mod + s;
                    if (row >= S) row -= S;
                    global_add_f64(SUp + k, (double)ring_get(t, lds, a.ring, b, q, row, nq, tid));
                }
            }
        }
#pragma unroll
        for (int l = 1; l < SNN_MAX_LAYERS; ++l) {
            if (l >= L) break;
            if (t.kind[l] != SNN_LIF) continue;
            const int li = t.lif[l];
            const int* ri = a.rec_idx + ((size_t)li * t.B + b) * (T + 1);
            const int k_lo = uniform32(ri[n]), k_hi = uniform32(ri[n + 1]);
            const size_t base = ((size_t)li * t.B + b) * t.cap;
            for (int kr = k_lo; kr < k_hi; ++kr) {
                const int i = uniform32(a.rec_n[base + kr]);
                for (int p = 0; p < t.P; ++p) {
                    if (t.pre[p] != l) continue;
                    const int q = t.post[p], nq = t.n[q];
                    if (tid >= nq) continue;
                    const size_t k = (size_t)i * nq + tid;
                    const int s = a.slot[t.woff[p] + k];
                    if (n + s <= T - 1) {
                        int row = n_mod + s;
                        if (row >= S) row -= S;
                        global_add_f64(a.SU + t.woff[p] + k,
                                       (double)ring_get(t, lds, a.ring, b, q, row, nq, tid));
                    }
                }
                if (i == tid) {
                    const float D = a.rec_D[base + kr];
                    if (D != 0.0f) lv[l] = __fadd_rn(lv[l], D);
                }
            }
        }
        n_mod = (n_mod == 0) ? S - 1 : n_mod - 1;
    }
}

struct FinalArgs {
    float* dW[SNN_MAXP];
    float* dD[SNN_MAXP];
    long long woff[SNN_MAXP + 1];
    int P;
    float tau_s, dt;
};

__global__ void finalize_kernel(const double* SU, const double* SD, FinalArgs a) {
    const long long g = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (g >= a.woff[a.P]) return;
    int p = 0;
    while (g >= a.woff[p + 1]) ++p;
    const long long k = g - a.woff[p];
    a.dW[p][k] = (float)(-(double)a.tau_s * SU[g]);
    a.dD[p][k] = (float)(-(double)a.dt * SD[g]);
}

__global__ void copy_state_kernel(const float* src, int stride, int off, int n, int B, float* dst) {
    const long long g = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (g >= (long long)B * n) return;
    const long long b = g / n, j = g % n;
    dst[g] = src[b * stride + off + j];
}

inline unsigned grid_for(long long n, int block) { return (unsigned)((n + block - 1) / block); }

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

hipError_t launch_forward(const FwdArgs& a, int threads, size_t lds, hipStream_t s) {
    hipLaunchKernelGGL(forward_kernel, dim3(a.t.B), dim3(threads), lds, s, a);
    return hipGetLastError();
}

hipError_t launch_loss(const float* z, const int* labels, const int* nstar, int B, int C, int loss,
                       float rscale, float tau_m, float* loss_out, float* src, const DevStatus* st,
                       hipStream_t s) {
    (void)nstar;
    hipLaunchKernelGGL(loss_kernel, dim3(1), dim3(256), 0, s, z, labels, B, C, loss, rscale, tau_m,
                       loss_out, src, st);
    return hipGetLastError();
}

hipError_t launch_fill_f64(double* p, long long n, hipStream_t s) {
    const unsigned g = (unsigned)std::min<long long>(grid_for(n, 256), 4096);
    hipLaunchKernelGGL(fill_f64_kernel, dim3(g > 0 ? g : 1), dim3(256), 0, s, p, n);
    return hipGetLastError();
}

hipError_t launch_backward_a(const BwdArgs& a, int threads, size_t lds, hipStream_t s) {
    hipLaunchKernelGGL(backward_a_kernel, dim3(a.t.B), dim3(threads), lds, s, a);
    return hipGetLastError();
}

hipError_t launch_backward_b(const BwdArgs& a, int threads, size_t lds, hipStream_t s) {
    hipLaunchKernelGGL(backward_b_kernel, dim3(a.t.B), dim3(threads), lds, s, a);
    return hipGetLastError();
}

hipError_t launch_finalize(const double* SU, const double* SD, float* const* dW, float* const* dD,
                           const long long* woff, const long long* cnt, int P, float tau_s, float dt,
                           hipStream_t s) {
    FinalArgs a{};
    for (int p = 0; p < P; ++p) {
        a.dW[p] = dW[p];
        a.dD[p] = dD[p];
        a.woff[p] = woff[p];
    }
    a.woff[P] = woff[P - 1] + cnt[P - 1];
    a.P = P;
    a.tau_s = tau_s;
    a.dt = dt;
    hipLaunchKernelGGL(finalize_kernel, dim3(grid_for(a.woff[P], 256)), dim3(256), 0, s, SU, SD, a);
    return hipGetLastError();
}

hipError_t launch_copy_state(const float* src, int stride, int off, int n, int B, float* dst,
                             hipStream_t s) {
    hipLaunchKernelGGL(copy_state_kernel, dim3(grid_for((long long)B * n, 256)), dim3(256), 0, s, src,
                       stride, off, n, B, dst);
    return hipGetLastError();
}

hipError_t set_kernel_lds_limits(size_t bytes) {
    hipError_t e;
    e = hipFuncSetAttribute((const void*)forward_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)bytes);
    if (e != hipSuccess) return e;
    e = hipFuncSetAttribute((const void*)backward_a_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)bytes);
    if (e != hipSuccess) return e;
    return hipFuncSetAttribute((const void*)backward_b_kernel,
                               hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
}
