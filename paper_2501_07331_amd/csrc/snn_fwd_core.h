// The LIF forward core of libsnn (gfx950, wave64), as a template; its
// instantiations for 256 and 1024 threads live in two sources so that they
// compile in parallel.  One workgroup per sample runs the LIF layers over T steps (Table 1, forward dynamics with delayed
// current jumps).  Lane j owns neuron j of every LIF layer and column j of
// every delay ring into that layer.
//
// Per step n: free dynamics, threshold and reset, wave ballots into LDS, one
// barrier, the delayed scatter of the spikes into the rings of the LIF-post
// projections, the spike records, and the arrivals (ring row n, projection
// by projection in projection order).  A ring cell sums its weights in emission
// order (step, then presynaptic neuron).
//
// Deferred scatter (rings in LDS, few zero-delay synapses): the weights and
// slots of step n's spikes are loaded during step n and scattered at step
// n + 1, so their load latency is hidden behind a whole step.  Arrivals with
// delay 0 cannot wait: every lane keeps, for each LIF-post projection, the
// presynaptic neurons with slot 0 into its post neuron (a bitmask in
// registers; their weights in LDS, in ascending presynaptic order) and adds
// those of step n's spikes to the arrival at step n, after the ring cell
// (which by then holds every earlier step's weights): the same fp32 sequence
// as adding in emission order.  With rings in HBM, more than two (layer,
// LIF-post projection) pairs, 1024 threads, no LDS left for the weights, or
// a post neuron with more than SNN_ZMAX zero-delay synapses, the scatter is
// immediate.
#pragma once

#include <type_traits>

#include "snn_device.h"

namespace {

constexpr int kZMax = SNN_ZMAX;   // zero-delay synapses per lane and projection

template <int MAXT, int NL, int NP, bool RL>
struct FwdCore {
    static constexpr int NWM = MAXT / 64;
    static constexpr int KP = (NL == 1) ? 8 : 4;     // spikes per step with prefetched weights
    static constexpr int KS = 4;                      // spikes per column_add_all of the deferred scatter
    // spikes per chunk of the immediate scatter: with rings in device memory
    // every chunk costs serialized round trips (weights, cells, stores), so
    // the chunks are larger there
    static constexpr int KI = RL ? KB : 16;
    static constexpr int NPA = NP > 0 ? NP : 1;
    // the deferred scatter's register lists fit without spills for one LIF
    // layer, or two with one LIF-post projection each, at 256 threads (and it
    // needs a ring to defer into)
    static constexpr bool kDeferable = RL && MAXT <= 256 && NP >= 1 && NL * NP <= 2;

    // Loads in flight for the next step: weights and slots of this step's
    // first KP spikes (this lane's post, every LIF-post projection) and the
    // next input arrival.
    struct Pre {
        uint2 ws[NL][NPA][KP];
        int cnt[NL];
        float ain;
    };

    struct Lane {
        float V[NL], I[NL];
        int cnt[NL];                          // records so far (exact; may pass the capacity)
        unsigned long long zb[NL][NPA][NWM];  // presynaptic neurons with slot 0 into this lane's post
    };

    template <typename Ptr>
    static __device__ __forceinline__ Ptr ring_col(const CoreFwdArgs& a, int b, int l, int pp, int col) {
        const FwdLayer& y = a.ly[l];
        if constexpr (RL) {
            return (lds_f32*)(reinterpret_cast<float*>(smem) + y.ring_lds[pp]) + col;
        } else {
            return (global_f32*)(y.ring[pp] + (size_t)b * (a.S + 1) * y.nq[pp]) + col;
        }
    }
    typedef typename std::conditional<RL, lds_f32*, global_f32*>::type RingPtr;

    static __device__ __forceinline__ __amdgpu_buffer_rsrc_t ws_rsrc(const CoreFwdArgs& a, int l, int pp) {
        const FwdLayer& y = a.ly[l];
        return __builtin_amdgcn_make_buffer_rsrc((void*)y.ws[pp], (short)0, y.npre[pp] * y.nq[pp] * 8,
                                                 0x00020000);
    }

    // Weights and slots of spikes ids[0 .. N) of layer l for this lane's post
    // of projection pp (rows clamped into the matrix; results of ids < 0 or of
    // unused projection entries are not used).
    template <int N>
    static __device__ __forceinline__ void load_ws(const CoreFwdArgs& a, int l, int pp, int tid,
                                                   const int (&ids)[N], uint2 (&w)[N]) {
        const FwdLayer& y = a.ly[l];
        const int nq = y.nq[pp], rmax = y.npre[pp] - 1;
        const __amdgpu_buffer_rsrc_t rs = ws_rsrc(a, l, pp);
        const int col8 = min(tid, nq - 1) * 8;
#pragma unroll
        for (int q = 0; q < N; ++q) {
            const int r = min(max(ids[q], 0), rmax);
            const auto v = __builtin_amdgcn_raw_buffer_load_b64(rs, col8, r * nq * 8, 0);
            w[q] = make_uint2((unsigned)v[0], (unsigned)v[1]);
        }
    }

    // Adds the weights of spikes 0 .. N) (valid below cnt) emitted at step e to
    // the ring cells of their arrivals, slots >= smin, arrivals before T, in
    // chunks of C.
    template <int N, int C>
    static __device__ __forceinline__ void scatter(const CoreFwdArgs& a, int b, int l, int pp, int tid,
                                                   int e, int cnt, int smin, const uint2 (&w)[N]) {
        const FwdLayer& y = a.ly[l];
        const int nq = y.nq[pp], S = a.S;
        const bool live = pp < y.npost && tid < nq;
        const int e_mod = e % S;
        RingPtr col = ring_col<RingPtr>(a, b, l, pp, min(tid, nq - 1));
#pragma unroll
        for (int q0 = 0; q0 < N; q0 += C) {
            if (cnt <= q0) continue;
            int row[C];
            float wv[C];
#pragma unroll
            for (int k = 0; k < C; ++k) {
                const int q = q0 + k;
                const int s = (int)w[q].y;
                int r = e_mod + s;
                r = (r >= S) ? r - S : r;
                const bool ok = live && q < cnt && s >= smin && e + s <= a.T - 1;
                row[k] = ok ? r : S;                  // row S: dummy
                wv[k] = __uint_as_float(w[q].x);
            }
            column_add_all(col, nq, row, wv);
        }
    }

    // All spikes of layer l at step e (mask words m), from position `from` on,
    // in chunks of KB with their weights loaded now.
    static __device__ __forceinline__ void scatter_rest(const CoreFwdArgs& a, int b, int l, int tid, int e,
                                        const unsigned long long (&m)[NWM],
                                        const unsigned long long* row, int from, int total,
                                        int smin) {
        const FwdLayer& y = a.ly[l];
        for (int q0 = from; q0 < total; q0 += KI) {
            int ids[KI];
            word_ids<NWM, KI>(m, row, a.NW, q0, ids);
#pragma unroll
            for (int pp = 0; pp < NP; ++pp) {
                if (pp >= y.npost) continue;
                uint2 w[KI];
                load_ws<KI>(a, l, pp, tid, ids, w);
                scatter<KI, KI>(a, b, l, pp, tid, e, total - q0, smin, w);
            }
        }
    }

    template <bool DEFER>
    static __device__ __forceinline__ void step(const CoreFwdArgs& a, int b, int tid, int n,
                                                const Pre& P, Pre& N, Lane& L) {
        const int lane = tid & 63, wave = tid >> 6;
        const int T = a.T, S = a.S, NW = a.NW;
        unsigned long long* masks = reinterpret_cast<unsigned long long*>(smem + a.mask_off);
        const int par = n % 3;

        // ---- free dynamics over one step, threshold, reset, ballots
        bool spk[NL];
#pragma unroll
        for (int l = 0; l < NL; ++l) {
            spk[l] = false;
            if (tid < a.ly[l].n) {
                const float gi = __fmul_rn(a.gamma, L.I[l]);
                const float Vm = __fmaf_rn(a.alpha, L.V[l], gi);
                L.I[l] = __fmul_rn(a.beta, L.I[l]);
                spk[l] = Vm >= a.theta;
                L.V[l] = spk[l] ? 0.0f : Vm;
            }
            const unsigned long long m = __ballot(spk[l]);
            if (lane == 0) masks[(size_t)(par * NL + l) * NW + wave] = m;
        }
        __syncthreads();

        // ---- counts, this lane's rank among the step's spikes (ascending
        // neuron order) and the step's first KP spikes
        unsigned long long mw[NL][NWM];
        int ids[NL][KP];
        int tot[NL], rank[NL], cnt0[NL];
#pragma unroll
        for (int l = 0; l < NL; ++l) {
            row_words<NWM>(masks + (size_t)(par * NL + l) * NW, NW, mw[l]);
            int before = 0, total = 0;
            unsigned long long own = 0;
#pragma unroll
            for (int w = 0; w < NWM; ++w) {
                const int c = __popcll(mw[l][w]);
                total += c;
                before += (w < wave) ? c : 0;
                own = (w == wave) ? mw[l][w] : own;
            }
            rank[l] = before + lanes_below(own);
            cnt0[l] = L.cnt[l];
            L.cnt[l] += total;
            tot[l] = total;
            word_ids<NWM, KP>(mw[l], masks + (size_t)(par * NL + l) * NW, NW, 0, ids[l]);
        }

        // loads issued a step ago (P) have landed; waiting here, not at the
        // step start, lets the dynamics, the barrier and the ids above cover
        // their latency (no stores of this step are in flight yet)
        __builtin_amdgcn_s_waitcnt(kWaitVm0);

        if constexpr (DEFER) {
            // ---- step n - 1's spikes into the rings (delays >= 1), weights loaded then
            if (n >= 1) {
#pragma unroll
                for (int l = 0; l < NL; ++l) {
#pragma unroll
                    for (int pp = 0; pp < NP; ++pp) {
                        if (pp < a.ly[l].npost)
                            scatter<KP, KS>(a, b, l, pp, tid, n - 1, P.cnt[l], 1, P.ws[l][pp]);
                    }
                    if (P.cnt[l] > KP) {
                        const unsigned long long* prow = masks + (size_t)(((n - 1) % 3) * NL + l) * NW;
                        unsigned long long mp[NWM];
                        row_words<NWM>(prow, NW, mp);
                        scatter_rest(a, b, l, tid, n - 1, mp, prow, KP, P.cnt[l], 1);
                    }
                }
            }
            // ---- loads for the next step: weights of this step's spikes
#pragma unroll
            for (int l = 0; l < NL; ++l) {
#pragma unroll
                for (int pp = 0; pp < NPA; ++pp) {
                    if (pp < NP) load_ws<KP>(a, l, pp, tid, ids[l], N.ws[l][pp]);
                }
                N.cnt[l] = tot[l];
            }
        } else {
            // ---- this step's spikes into the rings (all delays), loaded now
#pragma unroll
            for (int l = 0; l < NL; ++l)
                scatter_rest(a, b, l, tid, n, mw[l], masks + (size_t)(par * NL + l) * NW, 0, tot[l], 0);
        }
        N.ain = a.A_in[((size_t)b * T + min(n + 1, T - 1)) * a.n1 + min(tid, a.n1 - 1)];

        // ---- spike records (I- of this step), step table, overflow
#pragma unroll
        for (int l = 0; l < NL; ++l) {
            const FwdLayer& y = a.ly[l];
            int* row = y.steptab + ((size_t)b * T + n) * SNN_STEP_ROW;
            if (tid == 0) {
                // internal record indices never pass the capacity (the
                // caller's count stays exact)
                y.rec_idx[(size_t)b * (T + 1) + n] = min(cnt0[l], a.cap);
                row[0] = tot[l];
                row[1] = min(cnt0[l], a.cap);
            }
            if (spk[l]) {
                if (rank[l] < SNN_STEP_IDS) row[2 + rank[l]] = tid;
                const int pos = cnt0[l] + rank[l];
                if (pos < a.cap) {
                    const size_t r = (size_t)b * a.cap + pos;
                    y.rec_n[r] = tid;
                    y.rec_s[r] = n;
                    y.rec_I[r] = L.I[l];
                    y.out_step[r] = n;
                    y.out_neuron[r] = tid;
                }
            }
            if (tid == 0 && cnt0[l] + tot[l] > a.cap) a.st->overflow = 1;
        }

        // ---- arrivals at step n: per projection into the layer, in projection order
        const int n_mod = n % S;
        const int lanes = NW * 64;
#pragma unroll
        for (int l = 0; l < NL; ++l) {
            const FwdLayer& y = a.ly[l];
            if (tid >= y.n) continue;
#pragma unroll
            for (int e = 0; e < 2; ++e) {
                if (e >= y.nin) continue;
                float add;
                const int sl = y.in_l[e];
                if (sl < 0) {
                    add = P.ain;
                } else {
                    const int pp = y.in_pp[e];
                    RingPtr c = ring_col<RingPtr>(a, b, sl, pp, tid) + n_mod * y.n;
                    add = *c;
                    *c = 0.0f;
                    if constexpr (DEFER) {
                        // delay-0 arrivals of this step's spikes, ascending presynaptic index
#pragma unroll
                        for (int ll = 0; ll < NL; ++ll) {
                            if (ll != sl) continue;
#pragma unroll
                            for (int pq = 0; pq < NPA; ++pq) {
                                if (pq != pp) continue;
                                // weights of this lane's zero-delay synapses, ascending
                                const lds_f32* zw = (const lds_f32*)(reinterpret_cast<float*>(smem + a.zw_off)) +
                                                    (size_t)(ll * NPA + pq) * kZMax * lanes + tid;
                                int kbase = 0;
#pragma unroll
                                for (int w = 0; w < NWM; ++w) {
                                    const unsigned long long z = L.zb[ll][pq][w];
                                    unsigned long long h = mw[ll][w] & z;
                                    while (h) {
                                        const int bit = __builtin_ctzll(h);
                                        const int k = kbase + __popcll(z & ((1ull << bit) - 1ull));
                                        add = __fadd_rn(add, zw[k * lanes]);
                                        h &= h - 1;
                                    }
                                    kbase += __popcll(z);
                                }
                            }
                        }
                    }
                }
                L.I[l] = __fadd_rn(L.I[l], add);
            }
        }
    }

    template <bool DEFER>
    static __device__ __forceinline__ void run_steps(const CoreFwdArgs& a, int b, int tid, Lane& L) {
        Pre A, B;
#pragma unroll
        for (int l = 0; l < NL; ++l) A.cnt[l] = 0;
        A.ain = a.A_in[(size_t)b * a.T * a.n1 + min(tid, a.n1 - 1)];
        int n = 0;
        for (; n + 1 < a.T; n += 2) {
            step<DEFER>(a, b, tid, n, A, B, L);
            step<DEFER>(a, b, tid, n + 1, B, A, L);
        }
        if (n < a.T) step<DEFER>(a, b, tid, n, A, B, L);
        if constexpr (DEFER) {
            // the spikes of the last step arrive after T: nothing to scatter
        }
    }

    static __device__ __forceinline__ void run(const CoreFwdArgs& a) {
        if (a.st->bad_input) return;
        const int b = blockIdx.x, tid = threadIdx.x;
        const int S = a.S;
        // ---- zero the ring columns this lane owns (rows 0 .. S, row S: dummy)
#pragma unroll
        for (int l = 0; l < NL; ++l) {
#pragma unroll
            for (int pp = 0; pp < NP; ++pp) {
                const FwdLayer& y = a.ly[l];
                if (pp >= y.npost || tid >= y.nq[pp]) continue;
                RingPtr c = ring_col<RingPtr>(a, b, l, pp, tid);
                for (int r = 0; r <= S; ++r) c[r * y.nq[pp]] = 0.0f;
            }
        }
        Lane L;
#pragma unroll
        for (int l = 0; l < NL; ++l) {
            L.V[l] = 0.0f;
            L.I[l] = 0.0f;
            L.cnt[l] = 0;
        }
        bool defer = kDeferable && a.zw_off >= 0;
        if constexpr (kDeferable) {
            // ---- delay-0 synapses into this lane's post, per LIF-post
            // projection: bitmask in registers, weights in LDS ascending
            const int lanes = a.NW * 64;
            bool over = false;
#pragma unroll
            for (int l = 0; l < NL; ++l) {
#pragma unroll
                for (int pp = 0; pp < NPA; ++pp) {
#pragma unroll
                    for (int w = 0; w < NWM; ++w) L.zb[l][pp][w] = 0ull;
                    if (!defer) continue;
                    lds_f32* zw = (lds_f32*)(reinterpret_cast<float*>(smem + a.zw_off)) +
                                  (size_t)(l * NPA + pp) * kZMax * lanes + tid;
                    const FwdLayer& y = a.ly[l];
                    if (pp >= NP || pp >= y.npost) continue;
                    const int nq = y.nq[pp];
                    const bool live = tid < nq;
                    const __amdgpu_buffer_rsrc_t rs = ws_rsrc(a, l, pp);
                    const int col8 = min(tid, nq - 1) * 8;
                    int cnt = 0;
                    for (int i0 = 0; i0 < y.n; i0 += 8) {
                        uint2 e8[8];
#pragma unroll
                        for (int k = 0; k < 8; ++k) {
                            const auto v = __builtin_amdgcn_raw_buffer_load_b64(
                                rs, col8, min(i0 + k, y.n - 1) * nq * 8, 0);
                            e8[k] = make_uint2((unsigned)v[0], (unsigned)v[1]);
                        }
#pragma unroll
                        for (int k = 0; k < 8; ++k) {
                            const int i = i0 + k;
                            if (!live || i >= y.n || e8[k].y != 0u) continue;
#pragma unroll
                            for (int w = 0; w < NWM; ++w)
                                if (w == (i >> 6)) L.zb[l][pp][w] |= 1ull << (i & 63);
                            if (cnt < kZMax) zw[cnt * lanes] = __uint_as_float(e8[k].x);
                            ++cnt;
                        }
                    }
                    over = over || cnt > kZMax;
                }
            }
            // block-wide OR of `over` through mask row 2, which step 2 writes
            // first (after the barriers of steps 0 and 1)
            unsigned long long* vote =
                reinterpret_cast<unsigned long long*>(smem + a.mask_off) + (size_t)2 * NL * a.NW;
            const unsigned long long m = __ballot(over);
            if ((tid & 63) == 0) vote[tid >> 6] = m;
            __syncthreads();
            bool any = false;
            for (int w = 0; w < a.NW; ++w) any = any || vote[w] != 0ull;
            defer = defer && !any;
        } else {
            __syncthreads();
        }
        if constexpr (kDeferable) {
            if (defer) run_steps<true>(a, b, tid, L);
            else run_steps<false>(a, b, tid, L);
        } else {
            run_steps<false>(a, b, tid, L);
        }

        // ---- final state and record counts
#pragma unroll
        for (int l = 0; l < NL; ++l) {
            const FwdLayer& y = a.ly[l];
            if (tid < y.n) {
                a.Vf[(size_t)b * a.nstate + a.soff[l] + tid] = L.V[l];
                a.If[(size_t)b * a.nstate + a.soff[l] + tid] = L.I[l];
            }
            if (tid == 0) {
                y.rec_idx[(size_t)b * (a.T + 1) + a.T] = min(L.cnt[l], a.cap);
                y.rec_cnt[b] = min(L.cnt[l], a.cap);
                y.out_count[b] = L.cnt[l];
                atomicAdd(&a.st->layer_spikes[l], (unsigned long long)L.cnt[l]);
            }
        }
    }
};

template <int MAXT, int NL, int NP, bool RL>
__global__ void __launch_bounds__(MAXT) forward_core_kernel(CoreFwdArgs a) {
    FwdCore<MAXT, NL, NP, RL>::run(a);
}

template <int MAXT, int NL, int NP>
void launch_f3(const CoreFwdArgs& a, bool rl, int threads, size_t lds, hipStream_t s) {
    if (rl)
        hipLaunchKernelGGL((forward_core_kernel<MAXT, NL, NP, true>), dim3(a.B), dim3(threads), lds, s, a);
    else
        hipLaunchKernelGGL((forward_core_kernel<MAXT, NL, NP, false>), dim3(a.B), dim3(threads), lds, s, a);
}

// Launches the instantiation for n_lif LIF layers with at most np LIF-post
// projections each; false: no such instantiation.
template <int MAXT>
bool launch_ft(const CoreFwdArgs& a, int n_lif, int np, bool rl, int threads, size_t lds, hipStream_t s) {
    switch (n_lif * 4 + np) {
        case 4 + 0: launch_f3<MAXT, 1, 0>(a, rl, threads, lds, s); return true;
        case 4 + 1: launch_f3<MAXT, 1, 1>(a, rl, threads, lds, s); return true;
        case 8 + 1: launch_f3<MAXT, 2, 1>(a, rl, threads, lds, s); return true;
        case 8 + 2: launch_f3<MAXT, 2, 2>(a, rl, threads, lds, s); return true;
        case 12 + 1: launch_f3<MAXT, 3, 1>(a, rl, threads, lds, s); return true;
        case 12 + 2: launch_f3<MAXT, 3, 2>(a, rl, threads, lds, s); return true;
        case 16 + 1: launch_f3<MAXT, 4, 1>(a, rl, threads, lds, s); return true;
        case 16 + 2: launch_f3<MAXT, 4, 2>(a, rl, threads, lds, s); return true;
        default: return false;
    }
}

template <int M, bool R>
hipError_t set_lds_limits_t(size_t bytes, int* bad) {
    const void* fns[] = {
        (const void*)forward_core_kernel<M, 1, 0, R>, (const void*)forward_core_kernel<M, 1, 1, R>,
        (const void*)forward_core_kernel<M, 2, 1, R>, (const void*)forward_core_kernel<M, 2, 2, R>,
        (const void*)forward_core_kernel<M, 3, 1, R>, (const void*)forward_core_kernel<M, 3, 2, R>,
        (const void*)forward_core_kernel<M, 4, 1, R>, (const void*)forward_core_kernel<M, 4, 2, R>};
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

}  // namespace
