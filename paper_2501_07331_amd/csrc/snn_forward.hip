// Forward-pass kernels of libsnn (gfx950, wave64): validation, delay
// rounding, input arrivals, the LIF core, the LI readout and the loss.
#include "snn_device.h"

namespace {

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
    const float* W[SNN_MAXP];
    long long woff[SNN_MAXP + 1];
    int P, max_delay;
};

// Delays are integer multiples of the time step: rint (half to even), clamp.
// Also writes (weight bits, slot) pairs for one-load access to both.
__global__ void round_delays_kernel(RoundArgs a, uint8_t* slot, uint2* ws, DevStatus* st) {
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
        ws[g] = make_uint2(__float_as_uint(a.W[p][g - a.woff[p]]), (unsigned)s);
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
            int* row = a.steptab + (((size_t)li * t.B + b) * T + n) * SNN_STEP_ROW;
            if (tid == 0) {
                a.rec_idx[((size_t)li * t.B + b) * (T + 1) + n] = min(cnt[l], t.cap);
                row[0] = total;
                row[1] = min(cnt[l], t.cap);
            }
            if (spk[l]) {
                const int rank = before + lanes_below(mk[wave]);
                if (rank < SNN_STEP_IDS) row[2 + rank] = tid;
                const int pos = cnt[l] + rank;
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

hipError_t launch_round_delays(const float* const* D, const float* const* W, const long long* woff,
                               const long long* cnt, int P, int max_delay, uint8_t* slot, uint2* ws,
                               DevStatus* st, hipStream_t s) {
    RoundArgs a{};
    for (int p = 0; p < P; ++p) {
        a.D[p] = D[p];
        a.W[p] = W[p];
        a.woff[p] = woff[p];
    }
    a.woff[P] = woff[P - 1] + cnt[P - 1];
    a.P = P;
    a.max_delay = max_delay;
    hipLaunchKernelGGL(round_delays_kernel, dim3(grid_for(a.woff[P], 256)), dim3(256), 0, s, a, slot,
                       ws, st);
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

hipError_t launch_copy_state(const float* src, int stride, int off, int n, int B, float* dst,
                             hipStream_t s) {
    hipLaunchKernelGGL(copy_state_kernel, dim3(grid_for((long long)B * n, 256)), dim3(256), 0, s, src,
                       stride, off, n, B, dst);
    return hipGetLastError();
}

hipError_t set_forward_lds_limits(size_t bytes) {
    const void* fns[] = {(const void*)input_scan_kernel, (const void*)forward_core_kernel<256>,
                         (const void*)forward_core_kernel<1024>, (const void*)readout_forward_kernel};
    for (const void* f : fns) {
        const hipError_t e =
            hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}
