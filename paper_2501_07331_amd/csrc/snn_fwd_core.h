// The LIF forward core of libsnn (gfx950, wave64), as a template; its
// instantiations for 256 and 1024 threads live in two sources so that they
// compile in parallel.  One workgroup per sample runs the LIF layers over T steps (Table 1, forward dynamics with delayed
// current jumps).  Lane j owns neuron j of every LIF layer and column j of
// every delay ring into that layer.
//
// Per step n: free dynamics, threshold and reset, wave ballots into LDS, a
// barrier, every spike's neuron into the step's spike list in LDS at its
// rank, a second barrier, the delayed scatter of the spikes (ids from the
// list) into the rings of the LIF-post projections, the spike records, and
// the arrivals (ring row n, projection by projection in projection order).
// A ring cell sums its weights in emission order (step, then presynaptic
// neuron).
//
// The scatter of a step's spikes is immediate: in chunks, their weight rows
// are loaded and added to the ring cells of their arrivals (delay 0
// included) before the step's arrivals are read.  (A variant that loaded
// the weights a step ahead and scattered them one step later, adding
// zero-delay synapses from per-lane lists, was slower on gfx950 and is
// gone.)
//
// With RO, one more wave runs the leaky-integrator readout fed by a LIF
// layer, in its own loop with the core waves' two barriers per step: after
// the barriers of step n it reads that layer's spike list of step n,
// adds the spikes' readout weights to the ring cells of their arrivals (an
// LDS ring of S_out + 1 rows, emission order per cell) and runs the LI step
// n.  Its work overlaps the core waves' own scatter instead of following the
// core as a separate kernel.  (Running it one step behind, with the weights
// of a step loaded a step ahead, was slower: 1.41 against 1.33 ms on the
// 700-256rec-20 step.)
//
// The sample's record arrays are held in vector registers as device-memory
// pointers (gptr): as generic pointers their stores were flat ones, which
// count on the LDS counter too, so that the next LDS wait of the step waited
// for their write acknowledgements (1.23 against 1.16 ms).  (One more wave
// that staged the input arrivals in an LDS FIFO several steps ahead, so that
// the core never waited for their loads, was slower: 1.18 ms.)
#pragma once

#include <type_traits>

#include "snn_device.h"

namespace {

template <int MAXT, int NL, int NP, bool RL, bool RO, bool CL>
struct FwdCore {
    static_assert(!CL || (MAXT == 64 && RL && !RO), "cluster mode: 64 neurons a workgroup, LDS rings");
    static constexpr int NPA = NP > 0 ? NP : 1;
    // mask words of a layer: one per wave, or (cluster) one per workgroup
    static constexpr int NWM = CL ? SNN_MAX_NEURONS / 64 : MAXT / 64;
    // spikes per chunk of the scatter: with rings in device memory every
    // chunk costs serialized round trips (weights, cells, stores), so wide
    // layers, which carry tens of spikes per step, take larger chunks there;
    // so does a cluster's step, whose weight loads all go out together (a
    // lone wave has the registers)
    static constexpr int KI = CL ? (NL <= 2 ? 32 : 16) : (RL || MAXT <= 256) ? KB : 16;

    // Load in flight for the next step: its input arrival.
    struct Pre {
        float ain;
    };

    struct Lane {
        float V[NL], I[NL];
        int cnt[NL];                          // records so far (exact; may pass the capacity)
        int own[NL];                          // spikes of this lane's neuron
        // this sample's record arrays and step table: uniform, but held in
        // vector registers (in scalar ones, beside the kernel arguments the
        // step uses, they are spilled and reloaded lane by lane every step)
        gptr<int> rn[NL], rs[NL], on[NL], os[NL], tab[NL], idx[NL];
        gptr<float> rI[NL];
        gptr<const float> ain;                // this lane's column of the input arrivals [T][n_1]
        gptr<DevStatus> st;
    };

    static __device__ __forceinline__ void record_ptrs(const CoreFwdArgs& a, int b, int j, Lane& L) {
        L.ain = (gptr<const float>)(a.A_in + (size_t)b * a.T * a.n1 + min(j, a.n1 - 1));
        L.st = (gptr<DevStatus>)a.st;
        asm volatile("" : "+v"(L.ain), "+v"(L.st));
#pragma unroll
        for (int l = 0; l < NL; ++l) {
            const FwdLayer& y = a.ly[l];
            const size_t r0 = (size_t)b * a.cap;
            L.rn[l] = (gptr<int>)(y.rec_n + r0);
            L.rs[l] = (gptr<int>)(y.rec_s + r0);
            L.rI[l] = (gptr<float>)(y.rec_I + r0);
            L.on[l] = (gptr<int>)(y.out_neuron + r0);
            L.os[l] = (gptr<int>)(y.out_step + r0);
            L.tab[l] = (gptr<int>)(y.steptab + (size_t)b * a.T * SNN_STEP_ROW);
            L.idx[l] = (gptr<int>)(y.rec_idx + (size_t)b * (a.T + 1));
            asm volatile("" : "+v"(L.rn[l]), "+v"(L.rs[l]), "+v"(L.rI[l]), "+v"(L.on[l]), "+v"(L.os[l]),
                              "+v"(L.tab[l]), "+v"(L.idx[l]));
        }
    }

    template <typename Ptr>
    static __device__ __forceinline__ Ptr ring_col(const CoreFwdArgs& a, int b, int l, int pp, int col) {
        const FwdLayer& y = a.ly[l];
        if constexpr (RL) {
            return (lds_f32*)(reinterpret_cast<float*>(smem) + y.ring_lds[pp]) + col;
        } else {
            return (global_f32*)(y.ring[pp] + (size_t)b * (y.S[pp] + 1) * y.nq[pp]) + col;
        }
    }
    typedef typename std::conditional<RL, lds_f32*, global_f32*>::type RingPtr;

    static __device__ __forceinline__ __amdgpu_buffer_rsrc_t ws_rsrc(const CoreFwdArgs& a, int l, int pp) {
        const FwdLayer& y = a.ly[l];
        return __builtin_amdgcn_make_buffer_rsrc((void*)y.ws[pp], (short)0, y.npre[pp] * y.nq[pp] * 8,
                                                 0x00020000);
    }

    // Weights and slots of spikes ids[0 .. N) of layer l for post j of
    // projection pp (rows clamped into the matrix; results of ids < 0 or of
    // unused projection entries are not used).
    template <int N>
    static __device__ __forceinline__ void load_ws(const CoreFwdArgs& a, int l, int pp, int j,
                                                   const int (&ids)[N], uint2 (&w)[N]) {
        const FwdLayer& y = a.ly[l];
        const int nq = y.nq[pp], rmax = y.npre[pp] - 1;
        const __amdgpu_buffer_rsrc_t rs = ws_rsrc(a, l, pp);
        const int col8 = min(j, nq - 1) * 8;
#pragma unroll
        for (int q = 0; q < N; ++q) {
            const int r = min(max(ids[q], 0), rmax);
            const auto v = __builtin_amdgcn_raw_buffer_load_b64(rs, col8, r * nq * 8, 0);
            w[q] = make_uint2((unsigned)v[0], (unsigned)v[1]);
        }
    }

    // Adds the weights of spikes 0 .. N) (valid below cnt) emitted at step e to
    // the ring cells of their arrivals, arrivals before T, in chunks of C.
    // The lane's ring column is tid, of post j (the same but in cluster
    // mode, whose rings hold the workgroup's 64 columns).
    template <int N, int C>
    static __device__ __forceinline__ void scatter(const CoreFwdArgs& a, int b, int l, int pp, int tid,
                                                   int j, int e, int cnt, const uint2 (&w)[N]) {
        const FwdLayer& y = a.ly[l];
        const int nq = y.nq[pp], S = y.S[pp];
        const int rw = CL ? 64 : nq;                  // ring row width
        const bool live = pp < y.npost && j < nq;
        const int e_mod = e % S;
        RingPtr col = ring_col<RingPtr>(a, b, l, pp, CL ? tid : min(tid, nq - 1));
        int stride = rw;
        if constexpr (RL) {
            // lanes past the layer add every spike to row S (dummy) of their
            // column (outside cluster mode another lane's): stride 0 from that
            // cell
            col = live ? col : col + S * rw;
            stride = live ? rw : 0;
        }
#pragma unroll
        for (int q0 = 0; q0 < N; q0 += C) {
            if (cnt <= q0) continue;
            int row[C];
            float wv[C];
#pragma unroll
            for (int k = 0; k < C; ++k) {
                const int q = q0 + k;
                const int s = (int)w[q].y;
                if constexpr (RL) {
                    // slots below lim arrive before T (none past the count);
                    // a masked spike adds -0 (x + -0 = x exactly) to its own
                    // row, which no pending step shares
                    const int lim = (q < cnt) ? a.T - e : 0;
                    const unsigned r = (unsigned)(e_mod + s);
                    row[k] = (int)min(r, r - (unsigned)S);     // (e + s) mod S, as e_mod + s < 2 S
                    wv[k] = (s < lim) ? __uint_as_float(w[q].x) : -0.0f;
                } else {
                    int r = e_mod + s;
                    r = (r >= S) ? r - S : r;
                    const bool ok = q < cnt && e + s <= a.T - 1;
                    row[k] = (live && ok) ? r : S;    // row S: dummy
                    wv[k] = __uint_as_float(w[q].x);
                }
            }
            if constexpr (CL) {
                // a lone wave, whose every LDS latency is exposed: rounds of
                // 8 (four LDS round trips for 32 spikes; fp32 LDS atomics
                // would keep the order too but cost about 64 cycles each)
                column_add_rounds<8>(col, stride, row, wv);
            } else {
                column_add(col, stride, row, wv);
            }
        }
    }

    // Ids of spikes q0 .. q0 + N of layer l's list of the step in LDS (one
    // workgroup per sample), uniform; -1 past the step's count.  Reading them
    // costs one LDS round trip where finding them lane by lane in the mask
    // words costs about sixty vector instructions a chunk.
    template <int N>
    static __device__ __forceinline__ void list_ids(const CoreFwdArgs& a, int l, int q0, int total,
                                                    int (&ids)[N]) {
        const int* list = reinterpret_cast<const int*>(smem + a.ids_off) + l * a.NW * 64;
        const int last = a.NW * 64 - 1;
#pragma unroll
        for (int k = 0; k < N; ++k) {
            const int v = __builtin_amdgcn_readfirstlane(list[min(q0 + k, last)]);
            ids[k] = (q0 + k < total) ? v : -1;
        }
    }

    // All spikes of layer l at step e (mask words m), in chunks of KI with
    // their weights loaded now; outside cluster mode the chunk's ids come
    // from the step's list in LDS.
    static __device__ __forceinline__ void scatter_rest(const CoreFwdArgs& a, int b, int l, int tid,
                                                        int j, int e, const unsigned long long (&m)[NWM],
                                                        const unsigned long long* row, int total) {
        const FwdLayer& y = a.ly[l];
        for (int q0 = 0; q0 < total; q0 += KI) {
            int ids[KI];
            if constexpr (CL)
                word_ids<NWM, KI, CL>(m, row, a.NW, q0, ids);
            else
                list_ids<KI>(a, l, q0, total, ids);
#pragma unroll
            for (int pp = 0; pp < NP; ++pp) {
                if (pp >= y.npost) continue;
                uint2 w[KI];
                load_ws<KI>(a, l, pp, j, ids, w);
                scatter<KI, KI>(a, b, l, pp, tid, j, e, total - q0, w);
            }
        }
    }

    // Cluster mode: this workgroup's ballot masks m[l] of step n go out as
    // tagged 32-bit halves (word (l G + g) 2 + h of the step's exchange), and
    // the words of all G workgroups come back into the LDS mask rows of the
    // step (the same layout: a 64-bit mask word is its two halves).  false:
    // the wait gave up.
    static __device__ __forceinline__ bool exchange(const CoreFwdArgs& a, int c, int g, int n,
                                                    const unsigned long long (&m)[NL], unsigned* lds_rows) {
        const int lane = threadIdx.x & 63, G = a.cl.G, nw = 2 * NL * G;
        const unsigned tag = a.cl.tag0 + 2u * (unsigned)n;
        unsigned long long* X = a.cl.x + ((size_t)c * 2 + (n & 1)) * nw;
        if (lane < 2 * NL) {
            unsigned long long ml = m[0];
#pragma unroll
            for (int l = 1; l < NL; ++l) ml = ((lane >> 1) == l) ? m[l] : ml;
            cl_put(X + ((lane >> 1) * G + g) * 2 + (lane & 1), tag,
                   (lane & 1) ? (unsigned)(ml >> 32) : (unsigned)ml);
        }
        for (int k0 = 0; k0 < nw; k0 += 64) {
            const int k = k0 + lane;
            unsigned v;
            if (!cl_get(X, min(k, nw - 1), k < nw, tag, v, &a.st->cl_abort)) return false;
            if (k < nw) lds_rows[k] = v;
        }
        return true;
    }

    // ---- the fused readout wave (RO)

    // This lane's readout column in the LDS ring; lanes past C add to the
    // dummy row of column C - 1 (stride 0).
    static __device__ __forceinline__ lds_f32* ro_col(const CoreFwdArgs& a, int lane, int& stride) {
        const int C = a.ro_C;
        lds_f32* col = (lds_f32*)(smem + a.ro_off) + min(lane, C - 1);
        stride = (lane < C) ? C : 0;
        return (lane < C) ? col : col + a.ro_S * C;
    }

    // Readout weights of spikes ids[0 .. KB) of the feeding layer for this
    // lane's output (rows clamped into the matrix; entries past a step's
    // count are not used).
    static __device__ __forceinline__ void ro_load(const CoreFwdArgs& a, int lane, const int (&ids)[KB],
                                                   uint2 (&w)[KB]) {
        const int C = a.ro_C;
        const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
            (void*)a.ro_ws, (short)0, a.ro_nfeed * C * 8, 0x00020000);
        const int col8 = min(lane, C - 1) * 8, rmax = a.ro_nfeed - 1;
#pragma unroll
        for (int k = 0; k < KB; ++k) {
            const int r = min(max(ids[k], 0), rmax);
            const auto v = __builtin_amdgcn_raw_buffer_load_b64(rs, col8, r * C * 8, 0);
            w[k] = make_uint2((unsigned)v[0], (unsigned)v[1]);
        }
    }

    // Adds one chunk of step e's spikes (readout weights w, count left from
    // the chunk on `left`) to the ring cells of their arrivals.
    static __device__ __forceinline__ void ro_add(const CoreFwdArgs& a, int e, int left,
                                                  const uint2 (&w)[KB], lds_f32* col, int stride) {
        const int S = a.ro_S, e_mod = e % S;
        int rw[KB];
        float wv[KB];
#pragma unroll
        for (int k = 0; k < KB; ++k) {
            // slots below lim arrive before T (none past the count); a masked
            // spike adds -0 to its own row (x + -0 = x exactly)
            const int s = (int)w[k].y;
            const int lim = (k < left) ? a.T - e : 0;
            const unsigned r = (unsigned)(e_mod + s);
            rw[k] = (int)min(r, r - (unsigned)S);
            wv[k] = (s < lim) ? __uint_as_float(w[k].x) : -0.0f;
        }
        column_add(col, stride, rw, wv);
    }

    // Step e of the readout (after the step's barriers): the feeding layer's
    // spikes of step e (their count from the masks row `row`, their ids from
    // the step's list) into the ring, chunk by chunk, then the LI step with
    // the arrivals of row e.
    template <bool SUM>
    static __device__ __forceinline__ void ro_step(const CoreFwdArgs& a, int lane, int e,
                                                   const unsigned long long* row, LiState& q) {
        const int C = a.ro_C;
        unsigned long long mw[NWM];
        row_words<NWM>(row, a.NW, mw);
        int total = 0;
#pragma unroll
        for (int w = 0; w < NWM; ++w) total += __popcll(mw[w]);
        int stride;
        lds_f32* col = ro_col(a, lane, stride);
        for (int q0 = 0; q0 < total; q0 += KB) {
            int ids[KB];
            list_ids<KB>(a, a.ro_feed, q0, total, ids);
            uint2 w[KB];
            ro_load(a, lane, ids, w);
            ro_add(a, e, total - q0, w, col, stride);
        }
        // arrivals of step e (then the row is free for step e + S)
        float x = 0.0f;
        const int e_mod = e % a.ro_S;
        if (lane < C) {
            x = col[e_mod * C];
            col[e_mod * C] = 0.0f;
        }
        li_update<SUM>(a.alpha, a.beta, a.gamma, e, x, q);
    }

    // The readout wave's loop: two barriers per step, as the core waves' steps
    // (the branch is per wave, so every wave reaches every barrier); then the
    // results.
    template <bool SUM>
    static __device__ __forceinline__ void ro_run(const CoreFwdArgs& a, int b, int lane) {
        const unsigned long long* masks = reinterpret_cast<const unsigned long long*>(smem + a.mask_off);
        LiState q{};
        for (int n = 0; n < a.T; ++n) {
            __syncthreads();
            __syncthreads();                             // the step's spike lists are in
            ro_step<SUM>(a, lane, n, masks + (size_t)((n % 3) * NL + a.ro_feed) * a.NW, q);
        }
        ro_finish(a, b, lane, q);
    }

    static __device__ __forceinline__ void ro_finish(const CoreFwdArgs& a, int b, int lane,
                                                     const LiState& q) {
        const int C = a.ro_C;
        if (lane >= C) return;
        const bool sum = a.ro_loss == SNN_LOSS_CE_SUM;
        a.z[(size_t)b * C + lane] = sum ? __fmul_rn(a.ro_scale, q.acc) : q.best;
        a.nstar[(size_t)b * C + lane] = sum ? -1 : q.nst;
        a.Vf[(size_t)b * a.nstate + (a.nstate - C) + lane] = q.V;
        a.If[(size_t)b * a.nstate + (a.nstate - C) + lane] = q.I;
    }

    // Free dynamics over one step, threshold, reset and ballots of this
    // lane's neuron j in every LIF layer: spk[l], and the wave's masks m[l].
    static __device__ __forceinline__ void dynamics(const CoreFwdArgs& a, int j, Lane& L, bool (&spk)[NL],
                                                    unsigned long long (&m)[NL]) {
#pragma unroll
        for (int l = 0; l < NL; ++l) {
            spk[l] = false;
            if (j < a.ly[l].n) {
                const float gi = __fmul_rn(a.gamma, L.I[l]);
                const float Vm = __fmaf_rn(a.alpha, L.V[l], gi);
                L.I[l] = __fmul_rn(a.beta, L.I[l]);
                spk[l] = Vm >= a.theta;
                L.V[l] = spk[l] ? 0.0f : Vm;
            }
            m[l] = __ballot(spk[l]);
        }
    }

    // Spikes of every layer at the step (LDS mask rows `rows`), and this
    // lane's rank among them (ascending neuron order; the lane's mask word
    // wv: its wave's, or in cluster mode its workgroup's, with own bits m).
    static __device__ __forceinline__ void counts(const CoreFwdArgs& a, const unsigned long long* rows, int wv,
                                                  const unsigned long long (&m)[NL],
                                                  unsigned long long (&mw)[NL][NWM], int (&tot)[NL],
                                                  int (&rank)[NL], int (&cnt0)[NL], Lane& L) {
#pragma unroll
        for (int l = 0; l < NL; ++l) {
            row_words<NWM>(rows + (size_t)l * a.NW, a.NW, mw[l]);
            int before = 0, total = 0;
#pragma unroll
            for (int w = 0; w < NWM; ++w) {
                const int cw = __popcll(mw[l][w]);
                total += cw;
                before += (w < wv) ? cw : 0;
            }
            rank[l] = before + lanes_below(m[l]);
            cnt0[l] = L.cnt[l];
            L.cnt[l] += total;
            tot[l] = total;
        }
    }

    // Arrivals at step n: per projection into the layer, in projection order
    // (P.ain: the input projection's, loaded a step ahead); the lane's ring
    // column is tid, 64 wide in cluster mode.
    static __device__ __forceinline__ void arrivals(const CoreFwdArgs& a, int b, int tid, int j, int n,
                                                    const Pre& P, Lane& L) {
#pragma unroll
        for (int l = 0; l < NL; ++l) {
            const FwdLayer& y = a.ly[l];
            if (j >= y.n) continue;
#pragma unroll
            for (int e = 0; e < 2; ++e) {
                if (e >= y.nin) continue;
                float add;
                const int sl = y.in_l[e];
                if (sl < 0) {
                    add = P.ain;
                } else {
                    const int S = y.in_S[e], n_mod = n % S;
                    RingPtr rc;
                    if constexpr (RL)
                        rc = (lds_f32*)(reinterpret_cast<float*>(smem) + y.in_ring_lds[e]) + tid;
                    else
                        rc = (global_f32*)(y.in_ring[e] + (size_t)b * (S + 1) * y.n) + tid;
                    rc += n_mod * (CL ? 64 : y.n);
                    add = *rc;
                    *rc = 0.0f;
                }
                L.I[l] = __fadd_rn(L.I[l], add);
            }
        }
    }

    // Spike records of step n (neuron, step, I- of this step), the step
    // table row, the overflow flag.
    static __device__ __forceinline__ void records(const CoreFwdArgs& a, int g, int tid, int j, int n,
                                                   const bool (&spk)[NL], const int (&rank)[NL],
                                                   const int (&cnt0)[NL], const int (&tot)[NL], Lane& L) {
#pragma unroll
        for (int l = 0; l < NL; ++l) {
            gptr<int> row = L.tab[l] + n * SNN_STEP_ROW;
            if (tid == 0 && g == 0) {
                // internal record indices never pass the capacity (the
                // caller's count stays exact)
                L.idx[l][n] = min(cnt0[l], a.cap);
                row[0] = tot[l];
                row[1] = min(cnt0[l], a.cap);
            }
            if (spk[l]) {
                ++L.own[l];
                if (rank[l] < SNN_STEP_IDS) row[2 + rank[l]] = j;
                const int pos = cnt0[l] + rank[l];
                if (pos < a.cap) {
                    L.rn[l][pos] = j;
                    L.rs[l][pos] = n;
                    L.rI[l][pos] = L.I[l];
                    L.os[l][pos] = n;
                    L.on[l][pos] = j;
                }
            }
            if (tid == 0 && cnt0[l] + tot[l] > a.cap) L.st->overflow = 1;
        }
    }

    // One step n of one workgroup per sample.
    static __device__ __forceinline__ void step(const CoreFwdArgs& a, int b, int tid, int n, const Pre& P,
                                                Pre& N, Lane& L) {
        const int lane = tid & 63, wave = tid >> 6;
        const int T = a.T, NW = a.NW;
        unsigned long long* masks = reinterpret_cast<unsigned long long*>(smem + a.mask_off);
        const int par = n % 3;

        bool spk[NL];
        unsigned long long mine[NL];
        dynamics(a, tid, L, spk, mine);
        if (lane == 0) {
#pragma unroll
            for (int l = 0; l < NL; ++l) masks[(size_t)(par * NL + l) * NW + wave] = mine[l];
        }
        __syncthreads();

        unsigned long long mw[NL][NWM];
        int tot[NL], rank[NL], cnt0[NL];
        counts(a, masks + (size_t)par * NL * NW, wave, mine, mw, tot, rank, cnt0, L);
        // every spike's neuron at its rank in its layer's list of the step,
        // which all waves read after one more barrier
        int* lists = reinterpret_cast<int*>(smem + a.ids_off);
#pragma unroll
        for (int l = 0; l < NL; ++l)
            if (spk[l]) lists[l * NW * 64 + rank[l]] = tid;
        __syncthreads();

        // the input arrival loaded a step ago (P) has landed
        __builtin_amdgcn_s_waitcnt(kWaitVm0);

        // ---- this step's spikes into the rings (all delays)
#pragma unroll
        for (int l = 0; l < NL; ++l)
            scatter_rest(a, b, l, tid, tid, n, mw[l], masks + (size_t)(par * NL + l) * NW, tot[l]);
        N.ain = L.ain[min(n + 1, T - 1) * a.n1];

        records(a, 0, tid, tid, n, spk, rank, cnt0, tot, L);
        arrivals(a, b, tid, tid, n, P, L);
    }

    static __device__ __forceinline__ void run_steps(const CoreFwdArgs& a, int b, int tid, Lane& L) {
        Pre A, B;
        A.ain = L.ain[0];
        int n = 0;
        for (; n + 1 < a.T; n += 2) {
            step(a, b, tid, n, A, B, L);
            step(a, b, tid, n + 1, B, A, L);
        }
        if (n < a.T) step(a, b, tid, n, A, B, L);
    }

    // ---- cluster mode: wave 0 of a workgroup runs its 64 neurons of every
    // LIF layer (dynamics, the exchange, records, arrivals), wave 1 + r ring
    // r (the LIF-post projections of the LIF layers, in layer then
    // projection order): the step's spike ids of its source layer, their
    // weights for its 64 posts and the ordered adds.  The rings fill in
    // parallel on the CU's SIMDs, each from one wave in emission order.  Per
    // step two barriers: after the exchange (the masks are in LDS) and after
    // the adds (the rings hold the step's arrivals); a wait that gives up
    // raises an LDS flag before the first, and every wave returns after it.

    // A workgroup barrier over LDS only: this wave's LDS accesses complete,
    // its device-memory ones may stay in flight.
    static __device__ __forceinline__ void lds_barrier() {
        asm volatile("" ::: "memory");
        __builtin_amdgcn_s_waitcnt(0xC07F);       // lgkmcnt(0); vmcnt, expcnt at their maximum
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
    }

    // Ring r = (source layer l, its LIF-post projection pp) of this wave
    // (1 + r), r counted in layer then projection order; false: none.
    static __device__ __forceinline__ bool ring_of(const CoreFwdArgs& a, int r, int& rl, int& rpp) {
        int k = 0;
#pragma unroll
        for (int l = 0; l < NL; ++l)
#pragma unroll
            for (int pp = 0; pp < NP; ++pp)
                if (pp < a.ly[l].npost) {
                    if (k == r) {
                        rl = l;
                        rpp = pp;
                        return true;
                    }
                    ++k;
                }
        return false;
    }

    static __device__ __forceinline__ int* cl_flag(const CoreFwdArgs& a) {
        return reinterpret_cast<int*>(smem + a.mask_off + (size_t)3 * NL * a.NW * sizeof(unsigned long long));
    }

    // The neuron wave's step n.  false: the exchange gave up.
    static __device__ __forceinline__ bool step_cl(const CoreFwdArgs& a, int b, int c, int g, int lane,
                                                   int n, const Pre& P, Pre& N, Lane& L) {
        const int j = g * 64 + lane, T = a.T, NW = a.NW;
        unsigned long long* masks = reinterpret_cast<unsigned long long*>(smem + a.mask_off);
        const int par = n % 3;
        bool spk[NL];
        unsigned long long mine[NL];
        dynamics(a, j, L, spk, mine);
        const bool ok = exchange(a, c, g, n, mine, reinterpret_cast<unsigned*>(masks + (size_t)par * NL * NW));
        // the next step's input arrival goes out right after the exchange,
        // so that no load of this wave is in flight when the next exchange
        // waits for its own (a wait covers every older access)
        N.ain = L.ain[min(n + 1, T - 1) * a.n1];
        if (!ok && lane == 0) *cl_flag(a) = 1;
        lds_barrier();                                   // the masks of step n are in
        if (!ok) return false;
        unsigned long long mw[NL][NWM];
        int tot[NL], rank[NL], cnt0[NL];
        counts(a, masks + (size_t)par * NL * NW, g, mine, mw, tot, rank, cnt0, L);
        records(a, g, lane, j, n, spk, rank, cnt0, tot, L);
        lds_barrier();                                   // every ring holds step n's arrivals
        arrivals(a, b, lane, j, n, P, L);
        return true;
    }

    // A ring wave: every step, the spikes of its source layer in chunks of
    // KI, each chunk's weight loads issued together, then added in order.
    static __device__ __forceinline__ void ring_wave(const CoreFwdArgs& a, int b, int g, int lane, int l,
                                                     int pp) {
        const int j = g * 64 + lane;
        const unsigned long long* masks = reinterpret_cast<const unsigned long long*>(smem + a.mask_off);
        const int* flag = cl_flag(a);
        for (int n = 0; n < a.T; ++n) {
            lds_barrier();                               // the masks of step n are in
            if (*flag) return;
            const unsigned long long* row = masks + (size_t)((n % 3) * NL + l) * a.NW;
            unsigned long long mw[NWM];
            row_words<NWM>(row, a.NW, mw);
            int tot = 0;
#pragma unroll
            for (int w = 0; w < NWM; ++w) tot += __popcll(mw[w]);
            for (int q0 = 0; q0 < tot; q0 += KI) {
                int ids[KI];
                word_ids<NWM, KI, true>(mw, row, a.NW, q0, ids);
                uint2 w[KI];
                load_ws<KI>(a, l, pp, j, ids, w);
                scatter<KI, KI>(a, b, l, pp, lane, j, n, tot - q0, w);
            }
            lds_barrier();                               // every ring holds step n's arrivals
        }
    }

    static __device__ __forceinline__ void run_cl(const CoreFwdArgs& a) {
        const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
        int c, g;
        cluster_rank((int)blockIdx.x, a.cl.G, c, g);
        const int b = a.cl.b0 + c, j = g * 64 + lane;
        int rl = 0, rpp = 0;
        const bool ring = wave > 0 && ring_of(a, wave - 1, rl, rpp);
        if (ring) {
            // the ring's columns, rows 0 .. S (row S: dummy)
            lds_f32* rc = ring_col<lds_f32*>(a, b, rl, rpp, lane);
            for (int r = 0; r <= a.ly[rl].S[rpp]; ++r) rc[r * 64] = 0.0f;
        } else if (wave == 0 && lane == 0) {
            *cl_flag(a) = 0;
        }
        __syncthreads();
        if (wave > 0) {
            if (ring) ring_wave(a, b, g, lane, rl, rpp);
            return;
        }
        Lane L;
#pragma unroll
        for (int l = 0; l < NL; ++l) {
            L.V[l] = 0.0f;
            L.I[l] = 0.0f;
            L.cnt[l] = 0;
            L.own[l] = 0;
        }
        record_ptrs(a, b, j, L);
        Pre A, B;
        A.ain = L.ain[0];
        int n = 0;
        for (; n + 1 < a.T; n += 2) {
            if (!step_cl(a, b, c, g, lane, n, A, B, L)) return;
            if (!step_cl(a, b, c, g, lane, n + 1, B, A, L)) return;
        }
        if (n < a.T && !step_cl(a, b, c, g, lane, n, A, B, L)) return;
        finish(a, b, g, lane, j, L);
    }

    // Final state, spike counts per neuron, record counts.
    static __device__ __forceinline__ void finish(const CoreFwdArgs& a, int b, int g, int tid, int j,
                                                  const Lane& L) {
#pragma unroll
        for (int l = 0; l < NL; ++l) {
            const FwdLayer& y = a.ly[l];
            if (j < y.n) {
                a.Vf[(size_t)b * a.nstate + a.soff[l] + j] = L.V[l];
                a.If[(size_t)b * a.nstate + a.soff[l] + j] = L.I[l];
                // integer sums over the samples: exact in any order
                if (y.ncount && L.own[l]) atomicAdd(&y.ncount[j], L.own[l]);
            }
            if (tid == 0 && g == 0) {
                y.rec_idx[(size_t)b * (a.T + 1) + a.T] = min(L.cnt[l], a.cap);
                y.rec_cnt[b] = min(L.cnt[l], a.cap);
                y.out_count[b] = L.cnt[l];
                atomicAdd(&a.st->layer_spikes[l], (unsigned long long)L.cnt[l]);
            }
        }
    }

    static __device__ __forceinline__ void run(const CoreFwdArgs& a) {
        if (a.st->bad_input || (CL && a.st->cl_abort)) return;
        if constexpr (CL) {
            run_cl(a);
            return;
        }
        const int b = blockIdx.x, tid = threadIdx.x;
        // ---- zero the ring columns this lane owns (rows 0 .. S, row S: dummy)
#pragma unroll
        for (int l = 0; l < NL; ++l) {
#pragma unroll
            for (int pp = 0; pp < NP; ++pp) {
                const FwdLayer& y = a.ly[l];
                if (pp >= y.npost || tid >= y.nq[pp]) continue;
                RingPtr c = ring_col<RingPtr>(a, b, l, pp, tid);
                for (int r = 0; r <= y.S[pp]; ++r) c[r * y.nq[pp]] = 0.0f;
            }
        }
        Lane L;
#pragma unroll
        for (int l = 0; l < NL; ++l) {
            L.V[l] = 0.0f;
            L.I[l] = 0.0f;
            L.cnt[l] = 0;
            L.own[l] = 0;
        }
        record_ptrs(a, b, tid, L);
        if constexpr (RO) {
            if ((tid >> 6) == a.NW) {
                // the readout wave: its ring's columns, rows 0 .. S (row S:
                // dummy), then its own loop
                if ((tid & 63) < a.ro_C) {
                    lds_f32* c = (lds_f32*)(smem + a.ro_off) + (tid & 63);
                    for (int r = 0; r <= a.ro_S; ++r) c[r * a.ro_C] = 0.0f;
                }
                __syncthreads();
                if (a.ro_loss == SNN_LOSS_CE_SUM)
                    ro_run<true>(a, b, tid & 63);
                else
                    ro_run<false>(a, b, tid & 63);
                return;
            }
        }
        __syncthreads();
        run_steps(a, b, tid, L);
        finish(a, b, 0, tid, tid, L);
    }
};

// MAXT: the most LIF neurons per layer (threads of the core waves); with RO
// the workgroup has one more wave.  CL: cluster mode (MAXT = 64: the neuron
// wave, then one wave per ring).
template <int MAXT, int NL, int NP, bool RL, bool RO, bool CL = false>
__global__ void __launch_bounds__(CL ? 64 * (1 + NL * NP) : MAXT + (RO ? 64 : 0))
    forward_core_kernel(CoreFwdArgs a) {
    FwdCore<MAXT, NL, NP, RL, RO, CL>::run(a);
}

template <int MAXT, int NL, int NP>
void launch_f3(const CoreFwdArgs& a, bool rl, int threads, size_t lds, hipStream_t s) {
    constexpr bool ro = MAXT <= 256;       // a fused readout adds a wave (at most 1024 threads)
    if (ro && a.ro_C > 0) {
        if (rl)
            hipLaunchKernelGGL((forward_core_kernel<MAXT, NL, NP, true, ro>), dim3(a.B), dim3(threads), lds, s, a);
        else
            hipLaunchKernelGGL((forward_core_kernel<MAXT, NL, NP, false, ro>), dim3(a.B), dim3(threads), lds, s, a);
    } else {
        if (rl)
            hipLaunchKernelGGL((forward_core_kernel<MAXT, NL, NP, true, false>), dim3(a.B), dim3(threads), lds, s, a);
        else
            hipLaunchKernelGGL((forward_core_kernel<MAXT, NL, NP, false, false>), dim3(a.B), dim3(threads), lds, s, a);
    }
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

template <int M, bool R, bool O>
hipError_t set_lds_limits_t(size_t bytes, int* bad) {
    const void* fns[] = {
        (const void*)forward_core_kernel<M, 1, 0, R, O>, (const void*)forward_core_kernel<M, 1, 1, R, O>,
        (const void*)forward_core_kernel<M, 2, 1, R, O>, (const void*)forward_core_kernel<M, 2, 2, R, O>,
        (const void*)forward_core_kernel<M, 3, 1, R, O>, (const void*)forward_core_kernel<M, 3, 2, R, O>,
        (const void*)forward_core_kernel<M, 4, 1, R, O>, (const void*)forward_core_kernel<M, 4, 2, R, O>};
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
