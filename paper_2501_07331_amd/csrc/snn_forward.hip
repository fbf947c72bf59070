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
        st->reg_loss = 0.0;
        st->cl_abort = 0;
        for (int l = 0; l < SNN_MAX_LAYERS; ++l) st->layer_spikes[l] = 0;
    }
}

__global__ void clear_abort_kernel(DevStatus* st) {
    if (threadIdx.x == 0) st->cl_abort = 0;
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
        // four events per thread and round, their loads issued together
        const int nt = blockDim.x;
        for (int e0 = lo + (int)threadIdx.x; e0 < hi; e0 += 4 * nt) {
            int s[4], i[4], sp[4], ip[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int e = min(e0 + u * nt, hi - 1), ep = max(e - 1, lo);
                s[u] = step[e];
                i[u] = neuron[e];
                sp[u] = step[ep];
                ip[u] = neuron[ep];
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int e = e0 + u * nt;
                if (e >= hi) continue;
                if (s[u] < 0 || s[u] >= T || i[u] < 0 || i[u] >= n_in) bad = true;
                if (e > lo && (long long)s[u] * n_in + i[u] <= (long long)sp[u] * n_in + ip[u]) bad = true;
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
    int dmax[SNN_MAXP];
    int P;
};

// Delays are integer multiples of the time step: rint (half to even), clamp
// to [0, the projection's largest delay].  Also writes (weight bits, slot)
// pairs for one-load access to both.
__global__ void round_delays_kernel(RoundArgs a, uint8_t* slot, uint2* ws, DevStatus* st) {
    const long long g = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    bool clamped = false;
    if (g < a.woff[a.P]) {
        int p = 0;
        while (g >= a.woff[p + 1]) ++p;
        const float r = rintf(a.D[p][g - a.woff[p]]);
        int s;
        if (!(r >= 0.0f)) { s = 0; clamped = true; }            // negative or NaN
        else if (r > (float)a.dmax[p]) { s = a.dmax[p]; clamped = true; }
        else s = (int)r;
        slot[g] = (uint8_t)s;
        ws[g] = make_uint2(__float_as_uint(a.W[p][g - a.woff[p]]), (unsigned)s);
    }
    const unsigned long long m = __ballot(clamped);
    if ((threadIdx.x & 63) == 0 && m) atomicAdd(&st->clamped, (unsigned long long)__popcll(m));
}

// ------------------------------------------------------------------ input scan

// Workgroup = (sample b, block of 64 posts of layer 1), one wave; lane j owns
// post j.  The sample's input events stream by once, in emission order, in
// chunks of KB = 8, and each chunk's weights are added into an LDS ring of
// R = S + TB - 1 arrival steps (row m % R; row R: dummy).  Rows of steps
// before the first emission step of the next chunk are final (every later
// event arrives at its emission step or after): they go out as A_in rows and
// are cleared, at most two per chunk on the common path.  A chunk whose
// arrivals fit the ring from the first row not yet written out (its steps
// span less than TB past that row) is added at once; otherwise (a gap in the
// input, or a sparse chunk) the rows up to the chunk go out first and its
// events are added one by one, each after writing out the rows before it.  A
// ring cell sums in emission order (column_add_all keeps the order of equal
// rows).
//
// Loads run two chunks ahead: the ids and steps of a pair of chunks (one
// event per lane) at least two chunks before use, and the weights and slots
// of chunk c + 2 while chunk c is added, in three register sets (the loop
// body covers six chunks, so every set and pair vector has a fixed
// register).  A chunk writes out its final rows before issuing loads, so the
// wait at the next chunk start lets exactly the newest 8 operations (chunk
// c + 1's weights) stay in flight.  The common path writes out at most two
// rows per chunk and has no loop.
__global__ void __launch_bounds__(64) input_scan_kernel(InScanArgs a) {
    if (a.st->bad_input) return;
    const int n1 = a.n1, T = a.T, TB = a.TB, R = a.S + a.TB - 1;
    const int nblk = (n1 + 63) >> 6;
    const int b = blockIdx.x / nblk, jb = blockIdx.x - b * nblk;
    const int lane = threadIdx.x, j = jb * 64 + lane;
    const bool live = j < n1;
    const int jc = min(j, n1 - 1);
    lds_f32* ring = (lds_f32*)smem + lane;                      // [R + 1][64]
    for (int r = 0; r <= R; ++r) ring[r * 64] = 0.0f;
    global_f32* out = (global_f32*)(a.A_in + (size_t)b * T * n1 + jc);
    const int E0 = a.in_idx[(size_t)b * (T + 1)], E1 = a.in_idx[(size_t)b * (T + 1) + T];
    int f = 0, fr = 0;                                           // rows < f written out; fr = f % R
    auto flush_one = [&]() {
        const float v = ring[fr * 64];
        ring[fr * 64] = 0.0f;
        if (live) out[(size_t)f * n1] = v;
        ++f;
        fr = (fr + 1 == R) ? 0 : fr + 1;
    };
    auto flush_to = [&](int m) {
        while (f < m) flush_one();
    };
    if (E1 > E0) {
        const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
            (void*)a.ws0, (short)0, a.n_in * n1 * 8, 0x00020000);
        const int col8 = jc * 8, row8 = n1 * 8;
        // events e0 + q for lanes q < 2 KB (clamped to the last event): the
        // byte offset of the event's weight row, and its step
        auto load_pair = [&](int e0, int& rowv, int& stv) {
            const int e = min(e0 + (lane & (2 * KB - 1)), E1 - 1);
            rowv = a.in_neuron[e] * row8;
            stv = a.in_step[e];
        };
        auto load_ws = [&](int rowv, int u8, uint2 (&w)[KB]) {
#pragma unroll
            for (int q = 0; q < KB; ++q) {
                const int off = __builtin_amdgcn_readlane(rowv, u8 + q);
                const auto v = __builtin_amdgcn_raw_buffer_load_b64(rs, col8, off, 0);
                w[q] = make_uint2((unsigned)v[0], (unsigned)v[1]);
            }
        };
        // before the chunk of events e0 ..: write out up to two rows that are
        // final (steps before the chunk's first); issued before the next loads
        // so that the stores are never among the newest operations a chunk
        // start waits past
        auto flush_before = [&](int e0, int stv, int u8) {
            if (E1 - e0 <= 0) return;
            const int st0 = __builtin_amdgcn_readlane(stv, u8);
            if (f < st0) flush_one();
            if (f < st0) flush_one();
        };
        // chunk of events e0 .. e0 + KB - 1 (steps in lanes u8 .. u8 + KB - 1 of stv)
        auto add_chunk = [&](int e0, int stv, int u8, const uint2 (&w)[KB]) {
            const int nv = E1 - e0;                              // valid events (uniform)
            if (nv <= 0) return;
            int st[KB];
#pragma unroll
            for (int q = 0; q < KB; ++q) st[q] = __builtin_amdgcn_readlane(stv, u8 + q);
            const int last = __builtin_amdgcn_readlane(stv, u8 + min(nv, KB) - 1);   // last valid step
            if (last - f < TB) {
                int row[KB];
                float wv[KB];
#pragma unroll
                for (int q = 0; q < KB; ++q) {
                    const int s = (int)w[q].y;
                    // uniform parts: the ring row of arrival step st[q], and
                    // the slots that arrive before T (none past the end)
                    const int r0 = fr + (st[q] - f);
                    const int lim = (q < nv) ? T - st[q] : 0;
                    const unsigned r = (unsigned)(r0 + s);
                    // an event past the end or arriving at or after T adds
                    // -0 (x + -0 = x exactly, signed zeros included) to its
                    // row, which lies in the lane's own ring window
                    row[q] = (int)min(r, r - (unsigned)R);     // r mod R (r < 2 R)
                    wv[q] = (s < lim) ? __uint_as_float(w[q].x) : -0.0f;
                }
                column_add(ring, 64, row, wv);
            } else {
                // rare: events one by one, reloaded
                const int n = min(nv, KB);
                for (int q = 0; q < n; ++q) {
                    const int e = e0 + q;
                    const int stq = a.in_step[e];
                    flush_to(stq);
                    const auto v = __builtin_amdgcn_raw_buffer_load_b64(rs, col8, a.in_neuron[e] * row8, 0);
                    const int s = (int)v[1];
                    int r = fr + s;
                    r = (r >= R) ? r - R : r;
                    if (stq + s < T) ring[r * 64] = __fadd_rn(ring[r * 64], __uint_as_float((unsigned)v[0]));
                }
            }
        };
        // vmcnt(8): all but the newest eight operations (chunk c + 1's weight
        // loads) have landed
        constexpr int kWaitVm8 = 0x0F70 | 8;
        int rowX, stX, rowY, stY, rowZ, stZ;
        uint2 w0[KB], w1[KB], w2[KB];
        load_pair(E0, rowX, stX);
        load_pair(E0 + 2 * KB, rowY, stY);
        __builtin_amdgcn_s_waitcnt(kWaitVm0);
        load_ws(rowX, 0, w0);
        load_ws(rowX, KB, w1);
        // per chunk: wait, write out, next pair's ids, weights of chunk c + 2,
        // add chunk c; pairs X, Y, Z hold events e0 .., e0 + 16 .., e0 + 32 ..
        for (int e0 = E0; e0 < E1; e0 += 6 * KB) {
            __builtin_amdgcn_s_waitcnt(kWaitVm8);
            flush_before(e0, stX, 0);
            load_pair(e0 + 4 * KB, rowZ, stZ);
            load_ws(rowY, 0, w2);
            add_chunk(e0, stX, 0, w0);
            __builtin_amdgcn_s_waitcnt(kWaitVm8);
            flush_before(e0 + KB, stX, KB);
            load_ws(rowY, KB, w0);
            add_chunk(e0 + KB, stX, KB, w1);
            if (e0 + 2 * KB >= E1) break;
            __builtin_amdgcn_s_waitcnt(kWaitVm8);
            flush_before(e0 + 2 * KB, stY, 0);
            load_pair(e0 + 6 * KB, rowX, stX);
            load_ws(rowZ, 0, w1);
            add_chunk(e0 + 2 * KB, stY, 0, w2);
            __builtin_amdgcn_s_waitcnt(kWaitVm8);
            flush_before(e0 + 3 * KB, stY, KB);
            load_ws(rowZ, KB, w2);
            add_chunk(e0 + 3 * KB, stY, KB, w0);
            if (e0 + 4 * KB >= E1) break;
            __builtin_amdgcn_s_waitcnt(kWaitVm8);
            flush_before(e0 + 4 * KB, stZ, 0);
            load_pair(e0 + 8 * KB, rowY, stY);
            load_ws(rowX, 0, w0);
            add_chunk(e0 + 4 * KB, stZ, 0, w1);
            __builtin_amdgcn_s_waitcnt(kWaitVm8);
            flush_before(e0 + 5 * KB, stZ, KB);
            load_ws(rowX, KB, w1);
            add_chunk(e0 + 5 * KB, stZ, KB, w2);
        }
    }
    flush_to(T);
}

// ------------------------------------------------------------------ readout

template <bool SUM>
__device__ __forceinline__ void li_step(const Topo& t, int n, float x, LiState& q) {
    li_update<SUM>(t.alpha, t.beta, t.gamma, n, x, q);
}

// The LI layer over T steps of one lane's arrival column (step n at
// col[n * C]).  The arrivals are read in blocks of U steps, the next block's
// reads issued before the current block is run (two register blocks taking
// turns, so no copy waits for a read in flight); reads past the end take row
// T - 1 and are not used.
template <bool SUM, typename Ptr>
__device__ __forceinline__ void li_run(Ptr col, int C, int T, const Topo& t, LiState& q) {
    constexpr int U = 16;
    float xa[U], xb[U];
    auto load = [&](int n0, float (&x)[U]) {
#pragma unroll
        for (int u = 0; u < U; ++u) x[u] = col[(size_t)min(n0 + u, T - 1) * C];
    };
    auto run = [&](int n0, const float (&x)[U]) {
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (n0 + u < T) li_step<SUM>(t, n0 + u, x[u], q);
    };
    load(0, xa);
    for (int n0 = 0; n0 < T; n0 += 2 * U) {
        load(n0 + U, xb);
        run(n0, xa);
        if (n0 + U >= T) break;
        load(n0 + 2 * U, xa);
        run(n0 + U, xb);
    }
}

// One workgroup per sample.  Waves come in groups of OB = ceil(C / 64), lane
// k of a group owning output neuron k; group g builds rows [g W, (g + 1) W)
// of the arrival table [T + 1][C] (row T: dummy), scattering the records
// emitted in its rows or in the S - 1 steps before them, in emission order,
// so the groups work on disjoint rows in parallel.  Then group 0 runs the LI
// layer over the T steps.  table_lds >= 0: the table lives in LDS; else in
// global memory ([B][T + 1][C], sized by the host for this case).
__global__ void __launch_bounds__(1024) readout_forward_kernel(ReadoutArgs a) {
    const Topo& t = a.t;
    if (a.st->bad_input) return;
    const int b = blockIdx.x, tid = threadIdx.x;
    const int C = t.n[t.out_l], T = t.T;
    const int OB = (C + 63) >> 6, ngrp = max(1, (int)(blockDim.x >> 6) / OB);
    const int wave = tid >> 6, grp = wave / OB;
    const int k = (wave % OB) * 64 + (tid & 63);
    const int pa = t.pre[t.out_p];
    float* lds = reinterpret_cast<float*>(smem);
    const bool in_lds = a.table_lds >= 0;
    // lanes past C share column C - 1's dummy cell and touch nothing else
    const int kc = min(k, C - 1);
    lds_f32* lcol = (lds_f32*)(lds + (in_lds ? a.table_lds : 0)) + kc;
    global_f32* gcol = in_lds ? nullptr : (global_f32*)(a.table + (size_t)b * (T + 1) * C) + kc;
    if (pa != 0) {
        const int W = (T + ngrp - 1) / ngrp;
        const int m0 = min(T, grp * W), m1 = min(T, m0 + W);
        if (grp < ngrp && m0 < m1) {
            if (k < C) {
                for (int m = m0; m < m1; ++m) {
                    if (in_lds) lcol[m * C] = 0.0f; else gcol[m * C] = 0.0f;
                }
            }
            const size_t base = ((size_t)t.lif[pa] * t.B + b) * t.cap;
            const int* idx = a.rec_idx + ((size_t)t.lif[pa] * t.B + b) * (T + 1);
            const int e_lo = idx[max(0, m0 - (t.Sp[t.out_p] - 1))], e_hi = idx[m1];
            const int wsb = t.n[pa] * C * 8;
            if (in_lds)
                scatter_events(a.rec_n + base, a.rec_s + base, e_lo, e_hi, a.ws, wsb, C, k, k < C, m0, m1,
                               T - m0, lcol + m0 * C, C);
            else
                scatter_events(a.rec_n + base, a.rec_s + base, e_lo, e_hi, a.ws, wsb, C, k, k < C, m0, m1,
                               T - m0, gcol + (size_t)m0 * C, C);
        }
        __syncthreads();
    }
    if (grp != 0) return;
    if (k >= C) return;
    const global_f32* ain = (const global_f32*)(a.A_in + (size_t)b * T * C) + k;
    LiState q{};
    const bool sum = t.loss == SNN_LOSS_CE_SUM;
    if (pa == 0) {
        if (sum) li_run<true>(ain, C, T, t, q); else li_run<false>(ain, C, T, t, q);
    } else if (in_lds) {
        if (sum) li_run<true>(lcol, C, T, t, q); else li_run<false>(lcol, C, T, t, q);
    } else {
        if (sum) li_run<true>(gcol, C, T, t, q); else li_run<false>(gcol, C, T, t, q);
    }
    const float V = q.V, I = q.I, acc = q.acc, best = q.best;
    const int nst = q.nst;
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
// g / tau_m (max) in fp64, g = (softmax - onehot) / B rounded to fp32 first.
__global__ void loss_kernel(const float* z, const int* labels, int B, int C, int loss, float rscale,
                            float tau_m, float* loss_out, double* src, const DevStatus* st) {
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
            src[(size_t)b * C + k] = (loss == SNN_LOSS_CE_SUM)
                                         ? (double)rscale * (double)g / (double)tau_m
                                         : (double)g / (double)tau_m;
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

// Time-invariant MSE on first output spike times (SNN_LOSS_DMSE), one
// workgroup per sample: the first record of each output neuron (records are
// sorted by step, so the smallest index; an LDS atomic min is order-free),
// z = first step x dt in ms (T dt if none), then in fp64 and in neuron order
// L_b = 1/2 sum_{i != c} e_i^2, e_i = z_i - z_c - delta, and the jump terms
// dL/dt of the batch mean, e_i / B at the first spike of i != c and
// -sum_i e_i / B at that of c, written per record (0 elsewhere).
__global__ void __launch_bounds__(256) dmse_loss_kernel(const int* rec_cnt, const int* rec_s,
                                                        const int* rec_n, int cap, const int* labels,
                                                        int B, int C, int T, float dt, float delta,
                                                        float* z, float* loss_out, double* xlp,
                                                        const DevStatus* st) {
    __shared__ int first[1024];
    if (st->bad_input) return;
    const int b = blockIdx.x, tid = threadIdx.x;
    const int cnt = min(rec_cnt[b], cap);
    const size_t base = (size_t)b * cap;
    for (int k = tid; k < C; k += blockDim.x) first[k] = cap;
    __syncthreads();
    for (int r = tid; r < cnt; r += blockDim.x) {
        atomicMin(&first[rec_n[base + r]], r);
        xlp[base + r] = 0.0;
    }
    __syncthreads();
    for (int k = tid; k < C; k += blockDim.x) {
        const int n0 = (first[k] < cap) ? rec_s[base + first[k]] : T;
        z[(size_t)b * C + k] = (float)((double)n0 * (double)dt);
    }
    __syncthreads();
    if (tid != 0) return;
    const int c = labels[b];
    const float* zb = z + (size_t)b * C;
    double L = 0.0, sc = 0.0;
    for (int k = 0; k < C; ++k) {
        if (k == c) continue;
        const double e = (double)zb[k] - (double)zb[c] - (double)delta;
        L += 0.5 * e * e;
        sc += e;
        if (first[k] < cap) xlp[base + first[k]] = e / (double)B;
    }
    if (first[c] < cap) xlp[base + first[c]] = -sc / (double)B;
    loss_out[b] = (float)L;
}

// The batch mean of the per-sample losses, summed in sample order in fp64
// from the fp64 values the per-sample kernel rounded to fp32 (one thread).
__global__ void dmse_mean_kernel(const float* z, const int* labels, int B, int C, float delta,
                                 float* loss_out, const DevStatus* st) {
    if (st->bad_input || threadIdx.x != 0) return;
    double tot = 0.0;
    for (int b = 0; b < B; ++b) {
        const int c = labels[b];
        const float* zb = z + (size_t)b * C;
        double L = 0.0;
        for (int k = 0; k < C; ++k) {
            if (k == c) continue;
            const double e = (double)zb[k] - (double)zb[c] - (double)delta;
            L += 0.5 * e * e;
        }
        tot += L;
    }
    loss_out[B] = (float)(tot / (double)B);
}

__global__ void zero_ints_kernel(int* p, long long n) {
    const long long g = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (g < n) p[g] = 0;
}

// Spike-count regulariser (one workgroup of 256): the per-neuron jump term
// -rho (cbar - nu) / B and the penalty sum_l (rho_l / 2) sum_i (cbar_i -
// nu)^2, cbar the neuron's spikes per sample over the batch, in fp64; each
// thread sums a fixed strided set of neurons, then a fixed-order tree.
__global__ void __launch_bounds__(256) spike_reg_kernel(RegArgs a) {
    __shared__ double part[256];
    if (a.st->bad_input) return;
    const int tid = threadIdx.x;
    double acc = 0.0;
    for (int l = 0; l < a.nl; ++l) {
        if (a.rho[l] == 0.0) continue;
        for (int i = tid; i < a.n[l]; i += 256) {
            const double e = (double)a.ncount[l][i] / (double)a.B - a.nu;
            a.nterm[l][i] = -a.rho[l] * e / (double)a.B;
            acc += 0.5 * a.rho[l] * e * e;
        }
    }
    part[tid] = acc;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if (tid < w) part[tid] += part[tid + w];
        __syncthreads();
    }
    if (tid == 0) a.st->reg_loss = part[0];
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

hipError_t launch_clear_abort(DevStatus* st, hipStream_t s) {
    hipLaunchKernelGGL(clear_abort_kernel, dim3(1), dim3(64), 0, s, st);
    return hipGetLastError();
}

hipError_t launch_validate(const int* off, const int* step, const int* neuron, int nnz, int B, int T,
                           int n_in, const int* labels, int C, DevStatus* st, hipStream_t s) {
    hipLaunchKernelGGL(validate_kernel, dim3(B), dim3(1024), 0, s, off, step, neuron, nnz, B, T, n_in,
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
                               const long long* cnt, int P, const int* dmax, uint8_t* slot, uint2* ws,
                               DevStatus* st, hipStream_t s) {
    RoundArgs a{};
    for (int p = 0; p < P; ++p) {
        a.D[p] = D[p];
        a.W[p] = W[p];
        a.woff[p] = woff[p];
        a.dmax[p] = dmax[p];
    }
    a.woff[P] = woff[P - 1] + cnt[P - 1];
    a.P = P;
    hipLaunchKernelGGL(round_delays_kernel, dim3(grid_for(a.woff[P], 256)), dim3(256), 0, s, a, slot,
                       ws, st);
    return hipGetLastError();
}

hipError_t launch_input_scan(const InScanArgs& a, size_t lds, hipStream_t s) {
    const int nblk = (a.n1 + 63) / 64;
    if (a.TB < 1 || a.S + a.TB - 1 < 1) return hipErrorInvalidValue;
    hipLaunchKernelGGL(input_scan_kernel, dim3(a.B * nblk), dim3(64), lds, s, a);
    return hipGetLastError();
}

hipError_t launch_readout_forward(const ReadoutArgs& a, int threads, size_t lds, hipStream_t s) {
    hipLaunchKernelGGL(readout_forward_kernel, dim3(a.t.B), dim3(threads), lds, s, a);
    return hipGetLastError();
}

hipError_t launch_loss(const float* z, const int* labels, int B, int C, int loss, float rscale,
                       float tau_m, float* loss_out, double* src, const DevStatus* st, hipStream_t s) {
    hipLaunchKernelGGL(loss_kernel, dim3(1), dim3(256), 0, s, z, labels, B, C, loss, rscale, tau_m,
                       loss_out, src, st);
    return hipGetLastError();
}

hipError_t launch_dmse_loss(const int* rec_cnt, const int* rec_s, const int* rec_n, int cap,
                            const int* labels, int B, int C, int T, float dt, float delta, float* z,
                            float* loss_out, double* xlp, const DevStatus* st, hipStream_t s) {
    if (C > 1024 || cap < 1) return hipErrorInvalidValue;
    hipLaunchKernelGGL(dmse_loss_kernel, dim3(B), dim3(256), 0, s, rec_cnt, rec_s, rec_n, cap, labels,
                       B, C, T, dt, delta, z, loss_out, xlp, st);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(dmse_mean_kernel, dim3(1), dim3(64), 0, s, z, labels, B, C, delta, loss_out, st);
    return hipGetLastError();
}

hipError_t launch_zero_ints(int* p, long long n, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(zero_ints_kernel, dim3(grid_for(n, 256)), dim3(256), 0, s, p, n);
    return hipGetLastError();
}

hipError_t launch_spike_reg(const RegArgs& a, hipStream_t s) {
    hipLaunchKernelGGL(spike_reg_kernel, dim3(1), dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_copy_state(const float* src, int stride, int off, int n, int B, float* dst,
                             hipStream_t s) {
    hipLaunchKernelGGL(copy_state_kernel, dim3(grid_for((long long)B * n, 256)), dim3(256), 0, s, src,
                       stride, off, n, B, dst);
    return hipGetLastError();
}

hipError_t set_forward_lds_limits(size_t bytes, int* bad) {
    const void* fns[] = {(const void*)input_scan_kernel, (const void*)readout_forward_kernel};
    for (int i = 0; i < (int)(sizeof(fns) / sizeof(fns[0])); ++i) {
        const hipError_t e =
            hipFuncSetAttribute(fns[i], hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
        if (e != hipSuccess) {
            if (bad) *bad = i;
            return e;
        }
    }
    return hipSuccess;
}

hipError_t launch_forward_core(const CoreFwdArgs& a, int n_lif, int threads, size_t lds,
                               hipStream_t s) {
    // the core waves, and one more for a fused readout (cores of up to 256 threads)
    const int core = 64 * a.NW;
    if (n_lif < 1 || n_lif > SNN_MAX_LIF || threads != core + (a.ro_C > 0 ? 64 : 0) ||
        (a.ro_C > 0 && (core > 256 || a.ro_C > 64 || a.ro_feed < 0 || a.ro_feed >= n_lif)))
        return hipErrorInvalidValue;
    int np = 0;
    bool rl = true;
    for (int l = 0; l < n_lif; ++l) {
        np = max(np, a.ly[l].npost);
        for (int pp = 0; pp < a.ly[l].npost; ++pp)
            if (a.ly[l].ring_lds[pp] < 0) rl = false;
    }
    const bool ok = (core <= 256) ? launch_forward_core_256(a, n_lif, np, rl, threads, lds, s)
                                  : launch_forward_core_1024(a, n_lif, np, rl, threads, lds, s);
    if (!ok) return hipErrorInvalidValue;
    return hipGetLastError();
}

hipError_t set_core_lds_limits(size_t bytes, int* bad) {
    hipError_t e = set_core_lds_limits_256(bytes, bad);
    if (e == hipSuccess) {
        e = set_core_lds_limits_1024(bytes, bad);
        if (e != hipSuccess && bad) *bad += 32;   // 1024-thread kernels: 32 .. 47
    }
    if (e == hipSuccess) {
        e = set_core_lds_limits_cl(bytes, bad);
        if (e != hipSuccess && bad) *bad += 48;   // cluster kernels: 48 ..
    }
    return e;
}
