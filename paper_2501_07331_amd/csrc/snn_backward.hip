// Backward-pass kernels of libsnn (gfx950, wave64): the readout adjoint, the
// LIF adjoint core, spike grouping and the weight / delay gradients (Table 1,
// backward dynamics and gradient updates; Methods, the lambda_V jump with
// delayed postsynaptic adjoints and the weight and delay gradients).
//
//  readout_adjoint  one workgroup per sample: the LI adjoints over reverse time
//                   (loss source only; a linear recursion, run in chunks of
//                   steps in three passes), their trajectories, then the
//                   readout part of the jump sum of every spike of the
//                   feeding layer, computed in parallel over the spikes.
//  backward_core    one workgroup per sample runs the LIF adjoints in reverse
//                   time.  The spikes of every step are known from the
//                   forward's per-step masks, so the weights and slots of a
//                   step's spikes, their I- and readout jump parts are
//                   loaded one step ahead; the per-step chain is then LDS and
//                   ALU work only: free dynamics, trajectory row, adjoint
//                   ring, delayed postsynaptic sums, one barrier, jumps.
//  group            spikes of every sample grouped by presynaptic neuron
//                   (counting sort and per-neuron sort in LDS).
//  gradients        workgroup = (post layer, block of J posts, block of
//                   samples): lanes over the presynaptic neurons of every
//                   projection into the layer; per sample the J post
//                   trajectories, the spike-list offsets and the spike steps
//                   are staged in LDS by direct loads, and each lane sums,
//                   over its spikes in step order, lambda_I and lambda_I -
//                   lambda_V at the delayed arrivals.  Sample blocks are
//                   reduced in a fixed order: no atomics, deterministic.
//
// The whole backward pass is fp64 (constants, adjoints, trajectories, rings,
// jump sums, gradient sums): the adjoints are amplified through small jump
// denominators I- - theta, and fp32 state there moves some gradients by
// percents from the exact (fp64) result on the audio-sized networks.
#include "snn_device.h"

namespace {

// ------------------------------------------------------------------ readout adjoint

// Per output k, over reverse time: lambda_I <- beta lambda_I + c lambda_V,
// lambda_V <- alpha lambda_V (old lambda_V in both), then the step's loss
// source; the values before the source are the trajectory.  The recursion is
// linear, so it runs in three passes over chunks of LC steps, a lane per
// (output, chunk): (A) each chunk from a zero state, (B) per output, the
// state entering each chunk, chunk by chunk from the top (the state after a
// whole chunk = M^LC (state entering it) + its zero-state response), (C)
// each chunk again from its entering state, writing the trajectory.  The
// chunk results pass through the trajectory array itself (the first row of
// each chunk, rewritten by C).  Then every thread takes spikes (n, i) of the
// feeding LIF layer: A2 = sum_k w_ik (lambda_V - lambda_I)_k at step n +
// slot_ik, over k ascending.  All fp64.
__global__ void __launch_bounds__(512) readout_adjoint_kernel(ReadoutBwdArgs a) {
    const int b = blockIdx.x, tid = threadIdx.x, nt = blockDim.x;
    const int C = a.C, T = a.T, LC = a.LC, nch = a.nch;
    lds_f64* tab = (lds_f64*)smem;                                // [T][C] lambda_I - lambda_V
    double2* trb = a.traj + (size_t)b * T * C;
    // every thread's first record (the spike pass below), loaded first
    const int cnt = a.rec_n ? a.rec_cnt[b] : 0;
    const size_t base = (size_t)b * a.cap;
    int i = 0, n = 0;
    if (tid < cnt) {
        i = a.rec_n[base + tid];
        n = a.rec_s[base + tid];
    }
    auto chunk = [&](int x, bool out) {
        const int k = x % C, c = x / C;
        const int lo = c * LC, hi = min(T, lo + LC) - 1;
        const double srcv = a.src[(size_t)b * C + k];
        const int nst = a.nstar[(size_t)b * C + k];
        double lI = 0.0, lv = 0.0;
        if (out) {
            const double2 e = trb[(size_t)lo * C + k];
            lI = e.x;
            lv = e.y;
        }
        for (int m = hi; m >= lo; --m) {
            if (m <= T - 2) {
                const double v = lv;
                lI = __dadd_rn(__dmul_rn(a.beta, lI), __dmul_rn(a.cc, v));
                lv = __dmul_rn(a.alpha, v);
            }
            if (out) {
                const double d = __dsub_rn(lI, lv);
                trb[(size_t)m * C + k] = make_double2(lI, d);
                if (a.tab_lds) tab[m * C + k] = d;
            }
            if (a.loss == SNN_LOSS_CE_SUM || nst == m) lv = __dsub_rn(lv, srcv);
        }
        if (!out) trb[(size_t)lo * C + k] = make_double2(lI, lv);
    };
    for (int x = tid; x < C * nch; x += nt) chunk(x, false);
    __syncthreads();
    for (int k = tid; k < C; k += nt) {
        double eI = 0.0, ev = 0.0;                                // entering the top chunk
        for (int c = nch - 1; c >= 0; --c) {
            double2* p = trb + (size_t)c * LC * C + k;
            const double2 r = *p;
            *p = make_double2(eI, ev);
            const double nI = __dadd_rn(__dadd_rn(__dmul_rn(a.P11, eI), __dmul_rn(a.P12, ev)), r.x);
            const double nv = __dadd_rn(__dmul_rn(a.P22, ev), r.y);
            eI = nI;
            ev = nv;
        }
    }
    __syncthreads();
    for (int x = tid; x < C * nch; x += nt) chunk(x, true);
    if (!a.rec_n) return;
    __syncthreads();
    for (int r = tid; r < cnt; r += nt) {
        // the next record's neuron and step, and the weights of this one in
        // chunks of 16 outputs, each chunk's loads issued before the last
        // chunk's terms are added (in output order)
        int i2 = 0, n2 = 0;
        if (r + nt < cnt) {
            i2 = a.rec_n[base + r + nt];
            n2 = a.rec_s[base + r + nt];
        }
        const uint2* wsr = a.ws + (size_t)i * C;
        uint2 e[16];
#pragma unroll
        for (int u = 0; u < 16; ++u) e[u] = wsr[min(u, C - 1)];
        double acc = 0.0;
        for (int k0 = 0; k0 < C; k0 += 16) {
            const bool more = k0 + 16 < C;
            uint2 f[16];
            if (more) {
#pragma unroll
                for (int u = 0; u < 16; ++u) f[u] = wsr[min(k0 + 16 + u, C - 1)];
            }
            double d[16];
#pragma unroll
            for (int u = 0; u < 16; ++u) {
                const int k = min(k0 + u, C - 1);
                const int m = min(n + (int)e[u].y, T - 1);
                d[u] = a.tab_lds ? (double)tab[m * C + k] : trb[(size_t)m * C + k].y;
            }
#pragma unroll
            for (int u = 0; u < 16; ++u)
                if (k0 + u < C && n + (int)e[u].y <= T - 1)
                    acc = __dsub_rn(acc, __dmul_rn((double)__uint_as_float(e[u].x), d[u]));
            if (more) {
#pragma unroll
                for (int u = 0; u < 16; ++u) e[u] = f[u];
            }
        }
        a.A2[base + r] = acc;
        i = i2;
        n = n2;
    }
}

// ------------------------------------------------------------------ backward core

// Row sums of four fp64 values per lane (a transposed butterfly within each
// 16-lane row: xor 1 and xor 2 exchange half of the values, xor 4 and xor 8
// the last one).  Afterwards lane row*16 + k, k < 4, holds the sum over the
// row of v[2 (k & 1) + (k >> 1)].
__device__ __forceinline__ double row_sum4(const double (&v)[4], int lane) {
    const bool b0 = lane & 1, b1 = lane & 2, b2 = lane & 4;
    double u[2];
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        const double send = b0 ? v[k] : v[k + 2];
        const double keep = b0 ? v[k + 2] : v[k];
        u[k] = keep + dpp_f64<0xB1>(send);             // quad_perm [1,0,3,2]: xor 1
    }
    const double send = b1 ? u[0] : u[1];
    const double keep = b1 ? u[1] : u[0];
    double x = keep + dpp_f64<0x4E>(send);             // quad_perm [2,3,0,1]: xor 2
    const double up = dpp_f64<0x104>(x);               // row_shl:4, from lane + 4
    const double dn = dpp_f64<0x114>(x);               // row_shr:4, from lane - 4
    x += b2 ? dn : up;
    x += dpp_f64<0x128>(x);                            // row_ror:8: xor 8
    return x;
}

// Loads in flight for the steps after the one being processed: the spike
// table row of step n - 1, and for step n everything the delayed sums and
// jumps need.  Spikes beyond KP in a step are loaded when they are processed.
template <int NL, int KP, int NPA>
struct BwdState {
    int cnt2[NL], ri2[NL];        // step n - 1: spikes, record index of the first
    int id2[NL][KP];              //   first KP spiking neurons (raw; valid for q < cnt2)
    int cnt3[NL], ri3[NL];        // step n
    int id3[NL][KP];
    uint2 ws[NL][NPA][KP];        //   (weight bits, slot) of the LIF-post projections, this lane's post
    int mine[NL];                 //   1 + position of this lane's neuron among id3[0 .. KP), 0: none
    float I[NL];                  //   I- (fp32 record) and extra jump numerator of this lane's spike
    double A2[NL];
};

template <int MAXT, int NL, int KP, int NP, bool RL>
struct BwdCore {
    static constexpr int NPA = NP > 0 ? NP : 1;
    static constexpr int ROW4 = (2 + KP + 3) / 4;      // int4 loads of a spike-table row
    typedef BwdState<NL, KP, NPA> State;

    // The sample's arrays: uniform, but held in vector registers (in scalar
    // ones, beside the kernel arguments the step uses, they are spilled and
    // reloaded lane by lane every step).
    struct Ptrs {
        double2* tr[NL];               // this lane's trajectory column (stride lif_total)
        const int* tab[NL];            // step table [T][SNN_STEP_ROW]
        const float* recI[NL];         // records [cap]
        const double* A2[NL];          // [cap], or NULL
        const int* recn[NL];
    };

    static __device__ __forceinline__ void make_ptrs(const CoreBwdArgs& a, int b, int tid, Ptrs& P) {
#pragma unroll
        for (int l = 0; l < NL; ++l) {
            const BwdLayer& y = a.ly[l];
            const size_t r0 = (size_t)b * a.cap;
            P.tr[l] = a.traj + (size_t)b * a.T * a.lif_total + y.lif_off + tid;
            P.tab[l] = y.steptab + (size_t)b * a.T * SNN_STEP_ROW;
            P.recI[l] = y.recI + r0;
            P.A2[l] = y.A2 ? y.A2 + r0 : nullptr;
            P.recn[l] = y.recn + r0;
            asm volatile("" : "+v"(P.tr[l]), "+v"(P.tab[l]), "+v"(P.recI[l]), "+v"(P.A2[l]), "+v"(P.recn[l]));
        }
    }

    // Spike-table row of step x: count, record index, first KP neurons.  The
    // row is the same for every lane, but its address carries a per-lane zero
    // that the compiler cannot see through: a load it knows to be uniform has
    // its result moved to scalar registers right where it lands, which would
    // wait for it there; these values are made scalar a step later, at use.
    static __device__ __forceinline__ void load_row(const int* tab, int x, int& cnt, int& ri,
                                                    int (&ids)[KP]) {
        int zero;
        asm volatile("v_mov_b32 %0, 0" : "=v"(zero));
        const int4* rp = reinterpret_cast<const int4*>(tab + x * SNN_STEP_ROW) + zero;
        int v[ROW4 * 4];
#pragma unroll
        for (int k = 0; k < ROW4; ++k) {
            const int4 e = rp[k];
            v[4 * k + 0] = e.x;
            v[4 * k + 1] = e.y;
            v[4 * k + 2] = e.z;
            v[4 * k + 3] = e.w;
        }
        cnt = v[0];
        ri = v[1];
#pragma unroll
        for (int q = 0; q < KP; ++q) ids[q] = v[2 + q];
    }

    // Weights, slots, own position, I- and A2 of a step's spikes ids[0 .. KP)
    // (valid for q < cnt; record index of ids[0] is ri + r0).  Only the
    // chunks of 4 that hold spikes are loaded; ids are made uniform so that
    // a row's address is scalar and the lane adds its column.
    static __device__ __forceinline__ void load_step(const CoreBwdArgs& a, const float* recI,
                                                     const double* A2p, int tid, int l, int ri, int cnt,
                                                     const int (&ids)[KP], int r0, uint2 (&ws)[NPA][KP],
                                                     int& mine, float& I, double& A2) {
        const BwdLayer& y = a.ly[l];
        // (the ids stay in vector registers: held in scalar ones, the 16 ids
        // and their row offsets overflow the scalar register file).  Entries
        // past the count are not ids (stale table entries): their loads are
        // bounds-checked buffer loads (an offset outside the matrix reads 0)
        // and their values are masked, so the ids are used unclamped.
        int idc[KP];
#pragma unroll
        for (int q = 0; q < KP; ++q) idc[q] = ids[q];
        mine = 0;
#pragma unroll
        for (int q0 = 0; q0 < KP; q0 += 4) {
            if (cnt <= q0) break;
#pragma unroll
            for (int pp = 0; pp < NP; ++pp) {
                const int nq = y.nq[pp];
                // rows past the entry's own (a stand-in entry may have fewer
                // than y.n) read as zero; such entries are masked anyway
                const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
                    (void*)y.ws[pp], (short)0, y.npre[pp] * nq * 8, 0x00020000);
                const int col8 = min(tid, nq - 1) * 8;
#pragma unroll
                for (int q = q0; q < q0 + 4; ++q) {
                    // (unsigned: a stale entry's offset wraps instead of overflowing)
                    const unsigned off = (unsigned)col8 + __umul24((unsigned)idc[q], (unsigned)(nq * 8));
                    const auto v = __builtin_amdgcn_raw_buffer_load_b64(rs, (int)off, 0, 0);
                    ws[pp][q] = make_uint2((unsigned)v[0], (unsigned)v[1]);
                }
            }
#pragma unroll
            for (int q = q0; q < q0 + 4; ++q)
                if (q < cnt && idc[q] == tid) mine = q + 1;
        }
        if (mine) {
            const int r = ri + r0 + mine - 1;
            I = recI[r];
            A2 = A2p ? A2p[r] : 0.0;
        }
    }

    // Issue the loads of B from A (processing step n).
    static __device__ __forceinline__ void advance(const CoreBwdArgs& a, const Ptrs& P, int tid, int n,
                                                   const State& A, State& B) {
#pragma unroll
        for (int l = 0; l < NL; ++l) {
            load_row(P.tab[l], max(n - 2, 0), B.cnt2[l], B.ri2[l], B.id2[l]);
            B.cnt3[l] = __builtin_amdgcn_readfirstlane(A.cnt2[l]);
            B.ri3[l] = __builtin_amdgcn_readfirstlane(A.ri2[l]);
#pragma unroll
            for (int q = 0; q < KP; ++q) B.id3[l][q] = A.id2[l][q];
            load_step(a, P.recI[l], P.A2[l], tid, l, B.ri3[l], B.cnt3[l], A.id2[l], 0, B.ws[l], B.mine[l],
                      B.I[l], B.A2[l]);
        }
    }

    // Delayed postsynaptic sums of spikes ids[q0 .. q0 + 4) (valid for q < cnt)
    // of layer l, reduced per 16-lane row into part_l[q][wave * 4 + row].
    // n_mod[pp]: n modulo the adjoint-ring slots of projection pp's post layer.
    static __device__ __forceinline__ void gather4(const CoreBwdArgs& a, int b, int tid, int n,
                                                   const int (&n_mod)[NPA], int l, int q0, int cnt,
                                                   const int (&ids)[KP], const uint2 (&ws)[NPA][KP],
                                                   double* part_l) {
        const BwdLayer& y = a.ly[l];
        const int lane = tid & 63, wave = tid >> 6;
        // the reads of the chunk, all in bounds (masked terms read row 0,
        // column 0), issued together; the empty asm takes them as operands so
        // that the compiler keeps them unconditional (it would otherwise move
        // each read behind its own mask branch and wait for it there) and one
        // wait covers all of them; a masked term is then +0
        double d[4][NPA];
        bool ok[4][NPA];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int q = q0 + k;
#pragma unroll
            for (int pp = 0; pp < NPA; ++pp) {
                d[k][pp] = 0.0;
                ok[k][pp] = false;
                if (pp >= NP) continue;
                const int nq = y.nq[pp], S = y.qS[pp];
                const int sq = (int)ws[pp][q].y;
                // uniform: slots below lim arrive by T - 1 (none past the
                // count or the projections); the row by an unsigned min, as
                // n_mod + sq < 2 S
                const int lim = (pp < y.npost && q < cnt) ? a.T - n : 0;
                const unsigned ru = (unsigned)(n_mod[pp] + sq);
                const int row = (int)min(ru, ru - (unsigned)S);
                ok[k][pp] = sq < lim && tid < nq;
                // (in LDS the row is always in the ring and the column is
                // clamped into it, so the read needs no mask; its value does)
                if (RL)
                    d[k][pp] = ((lds_f64*)(smem + y.qring_lds[pp]))[__umul24(row, nq) + min(tid, nq - 1)];
                else   // (masked reads share one line of device memory)
                    d[k][pp] = ((global_f64*)(y.qring[pp] +
                                              ((size_t)b * S + (ok[k][pp] ? row : 0)) * nq))[ok[k][pp] ? tid : 0];
            }
        }
        if constexpr (NPA == 1) {
            asm volatile("" : "+v"(d[0][0]), "+v"(d[1][0]), "+v"(d[2][0]), "+v"(d[3][0]));
        } else {
            asm volatile("" : "+v"(d[0][0]), "+v"(d[1][0]), "+v"(d[2][0]), "+v"(d[3][0]),
                              "+v"(d[0][1]), "+v"(d[1][1]), "+v"(d[2][1]), "+v"(d[3][1]));
        }
        double v[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int q = q0 + k;
            v[k] = 0.0;
#pragma unroll
            for (int pp = 0; pp < NP; ++pp) {
                // a masked term is +0 (v - 0 = v exactly)
                const double t = __dmul_rn((double)__uint_as_float(ws[pp][q].x), d[k][pp]);
                v[k] = __dsub_rn(v[k], ok[k][pp] ? t : 0.0);
            }
        }
        const double x = row_sum4(v, lane);
        const int k = lane & 15;
        if (k < 4) part_l[(size_t)(q0 + 2 * (k & 1) + (k >> 1)) * (4 * a.NW) + wave * 4 + (lane >> 4)] = x;
    }

    static __device__ __forceinline__ void gather(const CoreBwdArgs& a, int b, int tid, int n,
                                                  const int (&n_mod)[NPA], int l, int cnt,
                                                  const int (&ids)[KP], const uint2 (&ws)[NPA][KP],
                                                  double* part_l) {
#pragma unroll
        for (int q0 = 0; q0 < KP; q0 += 4)
            if (cnt > q0) gather4(a, b, tid, n, n_mod, l, q0, cnt, ids, ws, part_l);
    }

    // The lambda_V jump of this lane's spike at position q of a round.
    static __device__ __forceinline__ void jump(const CoreBwdArgs& a, const double* part_l, int q,
                                                float I, double A2, double& lv,
                                                unsigned long long& deg) {
        double A = A2;
        if (NP > 0) {
            const double* pq = part_l + (size_t)q * (4 * a.NW);
            double Ap = 0.0;
            if constexpr (MAXT <= 256) {
                // the 4 NW partials read together, then added in order
                constexpr int NPART = 4 * (MAXT / 64);
                const int np = 4 * a.NW;
                double pv[NPART];
#pragma unroll
                for (int i = 0; i < NPART; ++i) pv[i] = pq[min(i, np - 1)];
#pragma unroll
                for (int i = 0; i < NPART; ++i) Ap = (i < np) ? Ap + pv[i] : Ap;
            } else {
                for (int i = 0; i < 4 * a.NW; ++i) Ap += pq[i];
            }
            A += Ap;
        }
        // tau_m dV/dt just before the crossing is I- - theta (V- = theta)
        const double den = __dsub_rn((double)I, a.theta);
        if (den > 0.0) {
            lv = __dadd_rn(lv, __dadd_rn(__dmul_rn(a.theta, lv), A) / den);
        } else {
            ++deg;
        }
    }

    struct Lane {
        double lv[NL], lI[NL];
        unsigned long long deg;
        int rnd;
    };

    // One reverse-time step n with the loads of A, issuing those of B.
    static __device__ __forceinline__ void step(const CoreBwdArgs& a, const Ptrs& P, int b, int tid, int n,
                                                const State& A, State& B, Lane& L) {
        const int T = a.T, LT = a.lif_total;
        double* part = reinterpret_cast<double*>(smem + a.part_off);   // [2][NL][KP][4 NW]
        // n modulo the adjoint-ring slots of each post layer read by layer l
        int nm[NL][NPA];
#pragma unroll
        for (int l = 0; l < NL; ++l)
#pragma unroll
            for (int pp = 0; pp < NPA; ++pp) nm[l][pp] = (NP > 0) ? n % a.ly[l].qS[pp] : 0;

        // the loads issued one step ago (A) have landed: wait for them once,
        // here, so that no later use waits for this step's loads
        __builtin_amdgcn_s_waitcnt(kWaitVm0);
        advance(a, P, tid, n, A, B);

        // ---- adjoint free dynamics, trajectory, adjoint ring
#pragma unroll
        for (int l = 0; l < NL; ++l) {
            const BwdLayer& y = a.ly[l];
            if (tid >= y.n) continue;
            if (n <= T - 2) {
                const double v = L.lv[l];
                L.lI[l] = __dadd_rn(__dmul_rn(a.beta, L.lI[l]), __dmul_rn(a.cc, v));
                L.lv[l] = __dmul_rn(a.alpha, v);
            }
            const double d = __dsub_rn(L.lI[l], L.lv[l]);
            P.tr[l][(size_t)n * LT] = make_double2(L.lI[l], d);
            if (y.ring_lds == -2) continue;
            const int n_own = n % y.S;
            if (RL)
                ((lds_f64*)(smem + y.ring_lds))[n_own * y.n + tid] = d;
            else
                ((global_f64*)(y.ring + ((size_t)b * y.S + n_own) * y.n))[tid] = d;
        }

        // ---- round 0: the first KP spikes of every layer, prefetched
        {
            const int pb = L.rnd & 1;
            ++L.rnd;
            if (NP > 0) {
#pragma unroll
                for (int l = 0; l < NL; ++l) {
                    double* part_l = part + (size_t)(pb * NL + l) * KP * (4 * a.NW);
                    gather(a, b, tid, n, nm[l], l, A.cnt3[l], A.id3[l], A.ws[l], part_l);
                }
            }
            __syncthreads();
#pragma unroll
            for (int l = 0; l < NL; ++l) {
                if (!A.mine[l]) continue;
                const double* part_l = part + (size_t)(pb * NL + l) * KP * (4 * a.NW);
                jump(a, part_l, A.mine[l] - 1, A.I[l], A.A2[l], L.lv[l], L.deg);
            }
        }
        // ---- further rounds when a step has more than KP spikes
        int rounds = 1;
#pragma unroll
        for (int l = 0; l < NL; ++l) rounds = max(rounds, (A.cnt3[l] + KP - 1) / KP);
        for (int r = 1; r < rounds; ++r) {
            const int pb = L.rnd & 1;
            ++L.rnd;
            int mine[NL];
            float I[NL];
            double A2[NL];
#pragma unroll
            for (int l = 0; l < NL; ++l) {
                const BwdLayer& y = a.ly[l];
                const int cnt = A.cnt3[l] - r * KP;          // spikes left from this round on
                int ids[KP];
                const int capm = max(a.cap - 1, 0);
#pragma unroll
                for (int q = 0; q < KP; ++q) ids[q] = P.recn[l][min(max(A.ri3[l] + r * KP + q, 0), capm)];
                uint2 ws[NPA][KP];
                load_step(a, P.recI[l], P.A2[l], tid, l, A.ri3[l], cnt, ids, r * KP, ws, mine[l], I[l], A2[l]);
                double* part_l = part + (size_t)(pb * NL + l) * KP * (4 * a.NW);
                if (NP > 0) gather(a, b, tid, n, nm[l], l, cnt, ids, ws, part_l);
            }
            __syncthreads();
#pragma unroll
            for (int l = 0; l < NL; ++l) {
                if (!mine[l]) continue;
                const double* part_l = part + (size_t)(pb * NL + l) * KP * (4 * a.NW);
                jump(a, part_l, mine[l] - 1, I[l], A2[l], L.lv[l], L.deg);
            }
        }
    }

    static __device__ void run(const CoreBwdArgs& a) {
        const int b = blockIdx.x, tid = threadIdx.x;
        const int T = a.T;
        Lane L;
#pragma unroll
        for (int l = 0; l < NL; ++l) {
            L.lv[l] = 0.0;
            L.lI[l] = 0.0;
        }
        L.deg = 0;
        L.rnd = 0;
        Ptrs P;
        make_ptrs(a, b, tid, P);
        State A, B;
        // step T - 1's data and step T - 2's table row, before the loop
#pragma unroll
        for (int l = 0; l < NL; ++l) {
            load_row(P.tab[l], T - 1, A.cnt3[l], A.ri3[l], A.id3[l]);
            load_row(P.tab[l], max(T - 2, 0), A.cnt2[l], A.ri2[l], A.id2[l]);
            A.cnt3[l] = __builtin_amdgcn_readfirstlane(A.cnt3[l]);
            A.ri3[l] = __builtin_amdgcn_readfirstlane(A.ri3[l]);
            load_step(a, P.recI[l], P.A2[l], tid, l, A.ri3[l], A.cnt3[l], A.id3[l], 0, A.ws[l], A.mine[l],
                      A.I[l], A.A2[l]);
        }
        int n = T - 1;
        for (; n >= 1; n -= 2) {
            step(a, P, b, tid, n, A, B, L);
            step(a, P, b, tid, n - 1, B, A, L);
        }
        if (n == 0) step(a, P, b, tid, 0, A, B, L);
        if (L.deg) atomicAdd(&a.st->degenerate, L.deg);
    }
};

// RL: every adjoint ring lives in LDS (else every one in HBM).
template <int MAXT, int NL, int KP, int NP, bool RL>
__global__ void __launch_bounds__(MAXT) backward_core_kernel(CoreBwdArgs a) {
    BwdCore<MAXT, NL, KP, NP, RL>::run(a);
}

// ------------------------------------------------------------------ backward core, cluster mode

// Cluster mode (the LIF layers' adjoint rings exceed one workgroup's LDS): G
// workgroups per sample, workgroup g holding the adjoint-ring columns of its
// neurons [64 g, 64 g + 64) of every LIF layer.  Wave 0, the neuron wave,
// runs lambda of those neurons (free dynamics, trajectories, ring rows, the
// exchange, the jumps); wave 1 + r, one per LIF -> LIF projection r (source
// layers in order, then projection order), the delayed postsynaptic sums of
// the step's spikes of its source layer over the workgroup's 64 posts.  The
// spike data of every wave is prefetched three steps deep (count and first
// record, then the ids, then a gather wave's weights and slots), so a step
// waits for memory once.  The spikes of a step go in rounds of at most KC
// per layer (steps without spikes have none); per round two barriers (the
// ring rows are written or the previous round's shares read; the shares are
// written) and one exchange of the shares between the workgroups: slot k
// (the round's spikes of every layer, in layer order) goes out as two
// tagged halves of word pair k of the workgroup's block, and lane k adds the
// G shares of slot k in workgroup order, which also keeps any workgroup from
// publishing twice into a buffer the others still read.
typedef unsigned v4u __attribute__((ext_vector_type(4)));
constexpr int kSc1 = 16;        // buffer access cache policy: agent scope (sc1)

template <int NL, int NP>
struct BwdCluster {
    static_assert(NP > 0, "cluster mode serves layers with LIF -> LIF projections");
    static constexpr int KC = kClKC;
    static constexpr int NS = NL * KC;            // exchange slots of a round
    static constexpr int NWD = 2 * NS;            // words of a workgroup's block

    // The staging in LDS at cl_off: shares [NL NP][KC][4] (fp64), slot
    // totals [NS] (fp64), own positions [NL][64] (int), the abort flag.
    static __device__ __forceinline__ double* shares(const CoreBwdArgs& a) {
        return reinterpret_cast<double*>(smem + a.cl_off);
    }
    static __device__ __forceinline__ double* totals(const CoreBwdArgs& a) {
        return shares(a) + NL * NP * KC * 4;
    }
    static __device__ __forceinline__ int* positions(const CoreBwdArgs& a) {
        return reinterpret_cast<int*>(totals(a) + NS);
    }
    static __device__ __forceinline__ int* flag(const CoreBwdArgs& a) { return positions(a) + NL * 64; }

    // Barrier over LDS only (device-memory accesses may stay in flight).
    static __device__ __forceinline__ void lds_barrier() {
        asm volatile("" ::: "memory");
        __builtin_amdgcn_s_waitcnt(0xC07F);       // lgkmcnt(0); vmcnt, expcnt at their maximum
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
    }

    // The sample's arrays: uniform, but held in vector registers (in scalar
    // ones, beside the kernel arguments, they are spilled and reloaded lane
    // by lane every step).
    struct Ptrs {
        const int* tab[NL];            // step table [T][SNN_STEP_ROW]
        const int* recn[NL];           // records [cap]
        const float* recI[NL];
        const double* A2[NL];          // or NULL
        double2* tr[NL];               // this lane's trajectory column (stride lif_total)
    };

    static __device__ __forceinline__ void make_ptrs(const CoreBwdArgs& a, int b, int j, Ptrs& P) {
#pragma unroll
        for (int l = 0; l < NL; ++l) {
            const BwdLayer& y = a.ly[l];
            const size_t r0 = (size_t)b * a.cap;
            P.tab[l] = y.steptab + (size_t)b * a.T * SNN_STEP_ROW;
            P.recn[l] = y.recn + r0;
            P.recI[l] = y.recI + r0;
            P.A2[l] = y.A2 ? y.A2 + r0 : nullptr;
            P.tr[l] = a.traj + (size_t)b * a.T * a.lif_total + y.lif_off + j;
            asm volatile("" : "+v"(P.tab[l]), "+v"(P.recn[l]), "+v"(P.recI[l]), "+v"(P.A2[l]), "+v"(P.tr[l]));
        }
    }

    // Spike count and first record index of layer l at step x (a per-lane
    // zero in the address keeps the compiler from making the load scalar and
    // waiting for it where it lands).
    static __device__ __forceinline__ int2 load_cr(const Ptrs& P, int l, int x) {
        int zero;
        asm volatile("v_mov_b32 %0, 0" : "=v"(zero));
        return reinterpret_cast<const int2*>(P.tab[l] + x * SNN_STEP_ROW)[zero];
    }

    // Lane q: the neuron of spike q0 + q of a step with records [ri, ri +
    // cnt) (clamped into them; -1 for a step without spikes).
    static __device__ __forceinline__ int load_id(const CoreBwdArgs& a, const Ptrs& P, int l, int ri, int cnt,
                                                  int q0) {
        const int q = min(q0 + (int)(threadIdx.x & 63), max(cnt - 1, 0));
        const int idx = min(max(ri + q, 0), max(a.cap - 1, 0));
        return (cnt > 0 && a.cap > 0) ? P.recn[l][idx] : -1;
    }

    // Weights and slots of spikes q < KC (ids in lanes q of `ids`) for post
    // j of projection pp of layer l (rows clamped into the matrix).
    static __device__ __forceinline__ void load_ws(const CoreBwdArgs& a, int l, int pp, int j, int ids,
                                                   uint2 (&w)[KC]) {
        const BwdLayer& y = a.ly[l];
        const int nq = y.nq[pp], rmax = y.npre[pp] - 1;
        const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
            (void*)y.ws[pp], (short)0, y.npre[pp] * nq * 8, 0x00020000);
        const int col8 = min(j, nq - 1) * 8;
#pragma unroll
        for (int q = 0; q < KC; ++q) {
            const int r = min(max(__builtin_amdgcn_readlane(ids, q), 0), rmax);
            const auto v = __builtin_amdgcn_raw_buffer_load_b64(rs, col8, r * nq * 8, 0);
            w[q] = make_uint2((unsigned)v[0], (unsigned)v[1]);
        }
    }

    // Rounds of a step: the most ceil(count / KC) over the layers.
    static __device__ __forceinline__ int rounds_of(const int (&cnt)[NL]) {
        int r = 0;
#pragma unroll
        for (int l = 0; l < NL; ++l) r = max(r, (cnt[l] + KC - 1) / KC);
        return r;
    }

    // ---- a gather wave: projection pp of layer l (post layer: its adjoint
    // ring qring, S rows, 64 columns)

    // Prefetch state entering step n: every layer's spike count and first
    // record at n (uniform), loaded ones at n - 1 and n - 2, the ids of
    // layer l at n - 1 (loaded; lane q: spike q).
    struct GState {
        int cn[NL], rn[NL];
        int2 c1[NL], c2[NL];
        int i1;
    };

    // Step n with this step's weights wc (landed); issues step n - 1's into
    // wn.  false: the cluster gave up (the flag was raised).
    static __device__ __forceinline__ bool gstep(const CoreBwdArgs& a, const Ptrs& P, int g, int r, int l,
                                                 int pp, int n, GState& st, uint2 (&wc)[KC], uint2 (&wn)[KC]) {
        const int lane = threadIdx.x & 63, j = g * 64 + lane, T = a.T;
        const BwdLayer& y = a.ly[l];
        const int nq = y.nq[pp], S = y.qS[pp];
        const bool live = j < nq;
        lds_f64* ring = (lds_f64*)(smem + y.qring_lds[pp]) + lane;
        double* sh = shares(a) + (size_t)r * KC * 4;
        int cnt = 0, ri = 0;
#pragma unroll
        for (int m = 0; m < NL; ++m)
            if (m == l) {
                cnt = st.cn[m];
                ri = st.rn[m];
            }
        const int rounds = rounds_of(st.cn);
        const int n_mod = n % S;
        for (int rd = 0; rd < rounds; ++rd) {
            lds_barrier();                                       // ring rows in, shares free
            if (*flag(a)) return false;
            const int q0 = rd * KC, nr = min(max(cnt - q0, 0), KC);
            if (rd > 0 && nr > 0) {
                // spikes past the prefetched ones: ids, then weights, now
                const int idr = load_id(a, P, l, ri, cnt, q0);
                load_ws(a, l, pp, j, idr, wc);
            }
            // (unrolled over the KC slots, so that the weights stay in
            // registers; chunks past the round's spikes are skipped)
#pragma unroll
            for (int k0 = 0; k0 < KC; k0 += 4) {
                if (k0 >= nr) break;
                double d[4], v[4];
                bool ok[4];
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const int sq = (int)wc[k0 + k].y;
                    const int lim = (k0 + k < nr) ? T - n : 0;
                    const unsigned ru = (unsigned)(n_mod + sq);
                    const int row = (int)min(ru, ru - (unsigned)S);
                    ok[k] = sq < lim && live;
                    d[k] = ring[row * 64];
                }
                asm volatile("" : "+v"(d[0]), "+v"(d[1]), "+v"(d[2]), "+v"(d[3]));
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    // a masked term is +0 (0 - 0 = +0)
                    const double t = __dmul_rn((double)__uint_as_float(wc[k0 + k].x), d[k]);
                    v[k] = __dsub_rn(0.0, ok[k] ? t : 0.0);
                }
                const double x = row_sum4(v, lane);
                const int k = lane & 15;
                if (k < 4) sh[(size_t)(k0 + 2 * (k & 1) + (k >> 1)) * 4 + (lane >> 4)] = x;
            }
            lds_barrier();                                       // shares written
        }
        // the next loads, issued while the neuron wave exchanges: counts three
        // steps ahead, ids two, weights one
        int2 c3[NL];
#pragma unroll
        for (int m = 0; m < NL; ++m) c3[m] = load_cr(P, m, max(n - 3, 0));
        int i2 = 0;
#pragma unroll
        for (int m = 0; m < NL; ++m)
            if (m == l)
                i2 = load_id(a, P, l, __builtin_amdgcn_readfirstlane(st.c2[m].y),
                             __builtin_amdgcn_readfirstlane(st.c2[m].x), 0);
        if (n > 0) load_ws(a, l, pp, j, st.i1, wn);
#pragma unroll
        for (int m = 0; m < NL; ++m) {
            st.cn[m] = __builtin_amdgcn_readfirstlane(st.c1[m].x);
            st.rn[m] = __builtin_amdgcn_readfirstlane(st.c1[m].y);
            st.c1[m] = st.c2[m];
            st.c2[m] = c3[m];
        }
        st.i1 = i2;
        return true;
    }

    static __device__ void gather_wave(const CoreBwdArgs& a, int b, int g, int r, int l, int pp) {
        const int j = g * 64 + (int)(threadIdx.x & 63), T = a.T;
        Ptrs P;
        make_ptrs(a, b, j, P);
        GState st;
        int2 c0[NL];
#pragma unroll
        for (int m = 0; m < NL; ++m) {
            c0[m] = load_cr(P, m, T - 1);
            st.c1[m] = load_cr(P, m, max(T - 2, 0));
            st.c2[m] = load_cr(P, m, max(T - 3, 0));
        }
        __builtin_amdgcn_s_waitcnt(kWaitVm0);
        int i0 = 0;
#pragma unroll
        for (int m = 0; m < NL; ++m) {
            st.cn[m] = __builtin_amdgcn_readfirstlane(c0[m].x);
            st.rn[m] = __builtin_amdgcn_readfirstlane(c0[m].y);
            if (m == l) {
                i0 = load_id(a, P, l, st.rn[m], st.cn[m], 0);
                st.i1 = load_id(a, P, l, __builtin_amdgcn_readfirstlane(st.c1[m].y),
                                __builtin_amdgcn_readfirstlane(st.c1[m].x), 0);
            }
        }
        __builtin_amdgcn_s_waitcnt(kWaitVm0);
        uint2 wa[KC], wb[KC];
        load_ws(a, l, pp, j, i0, wa);
        int n = T - 1;
        for (; n >= 1; n -= 2) {
            if (!gstep(a, P, g, r, l, pp, n, st, wa, wb)) return;
            if (!gstep(a, P, g, r, l, pp, n - 1, st, wb, wa)) return;
        }
        if (n == 0) gstep(a, P, g, r, l, pp, 0, st, wa, wb);
    }

    // ---- the neuron wave

    // Exchange of one round: K slots (uniform).  false: the wait gave up.
    static __device__ __forceinline__ bool exchange(const CoreBwdArgs& a, int c, int g, int rnd, int K,
                                                    const int (&off)[NL], const int (&nr)[NL],
                                                    const int (&rof)[NL], const int (&nring)[NL]) {
        const int lane = threadIdx.x & 63, G = a.cl.G;
        const unsigned tag = a.cl.tag0 + 2u * (unsigned)rnd;
        unsigned long long* X = a.cl.x + ((size_t)c * 2 + (rnd & 1)) * (size_t)G * NWD;
        const __amdgpu_buffer_rsrc_t rs =
            __builtin_amdgcn_make_buffer_rsrc((void*)X, (short)0, G * NWD * 8, 0x00020000);
        const double* sh = shares(a);
        double* tot = totals(a);
        for (int k0 = 0; k0 < K; k0 += 64) {
            const int k = k0 + lane;
            const bool mine = k < K;
            // this workgroup's share of slot k: its projections' four row
            // partials, each added in order, projections in order
            if (mine) {
                int l = 0;
#pragma unroll
                for (int m = 1; m < NL; ++m) l = (k >= off[m]) ? m : l;
                int q = k, rr = 0, nrg = 0;
#pragma unroll
                for (int m = 0; m < NL; ++m)
                    if (m == l) {
                        q = k - off[m];
                        rr = rof[m];
                        nrg = nring[m];
                    }
                double v = 0.0;
                for (int p = 0; p < nrg; ++p) {
                    const double* pq = sh + ((size_t)(rr + p) * KC + q) * 4;
                    v += ((pq[0] + pq[1]) + pq[2]) + pq[3];
                }
                // both tagged halves in one 16-byte agent-scope store
                const unsigned long long u = (unsigned long long)__double_as_longlong(v);
                const v4u wd = {(unsigned)u, tag, (unsigned)(u >> 32), tag};
                __builtin_amdgcn_raw_buffer_store_b128(wd, rs, (g * NWD + 2 * k) * 8, 0, kSc1);
            }
            // every workgroup's share of slot k, added in workgroup order: one
            // 16-byte load per workgroup (each 8-byte half single-copy atomic
            // with its own tag; a torn pair is read again)
            unsigned need = mine ? (unsigned)((1ull << G) - 1) : 0u;
            unsigned lo[SNN_MAX_NEURONS / 64], hi[SNN_MAX_NEURONS / 64];
            const int kk = 2 * min(k, K - 1);
            for (int spin = 0;; ++spin) {
                asm volatile("" ::: "memory");               // the loads are issued anew every poll
                v4u wv[SNN_MAX_NEURONS / 64];
#pragma unroll
                for (int i = 0; i < SNN_MAX_NEURONS / 64; ++i)
                    if ((need >> i) & 1u) wv[i] = __builtin_amdgcn_raw_buffer_load_b128(rs, (i * NWD + kk) * 8, 0, kSc1);
#pragma unroll
                for (int i = 0; i < SNN_MAX_NEURONS / 64; ++i)
                    if (((need >> i) & 1u) && wv[i].y == tag && wv[i].w == tag) {
                        lo[i] = wv[i].x;
                        hi[i] = wv[i].z;
                        need &= ~(1u << i);
                    }
                if (__ballot(need != 0) == 0) break;
                if ((spin & 255) == 255) {
                    if (__hip_atomic_load(&a.st->cl_abort, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) return false;
                    if (spin >= kClusterSpins) {
                        __hip_atomic_store(&a.st->cl_abort, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        return false;
                    }
                }
                __builtin_amdgcn_s_sleep(1);
            }
            if (mine) {
                double s = 0.0;
#pragma unroll
                for (int gp = 0; gp < SNN_MAX_NEURONS / 64; ++gp)
                    if (gp < G)
                        s += __longlong_as_double((long long)(((unsigned long long)hi[gp] << 32) | lo[gp]));
                tot[k] = s;
            }
        }
        return true;
    }

    static __device__ void neuron_wave(const CoreBwdArgs& a, int b, int c, int g) {
        const int lane = threadIdx.x & 63, j = g * 64 + lane, T = a.T, LT = a.lif_total;
        double lv[NL], lI[NL];
        unsigned long long deg = 0;
        int rnd = 0;
        // gather waves of each layer: the first one's index and how many
        int rof[NL], nring[NL];
        {
            int r = 0;
#pragma unroll
            for (int l = 0; l < NL; ++l) {
                rof[l] = r;
                nring[l] = a.ly[l].npost;
                r += a.ly[l].npost;
            }
        }
#pragma unroll
        for (int l = 0; l < NL; ++l) {
            lv[l] = 0.0;
            lI[l] = 0.0;
        }
        int* pos = positions(a);
        const double* tot = totals(a);
        Ptrs P;
        make_ptrs(a, b, j, P);
        // pipeline: (count, first record) of steps n, n - 1; ids of n
        int2 c0[NL], c1[NL];
        int id0[NL];
#pragma unroll
        for (int l = 0; l < NL; ++l) {
            c0[l] = load_cr(P, l, T - 1);
            c1[l] = load_cr(P, l, max(T - 2, 0));
        }
        __builtin_amdgcn_s_waitcnt(kWaitVm0);
        int cnt0[NL], ri0[NL];
#pragma unroll
        for (int l = 0; l < NL; ++l) {
            cnt0[l] = __builtin_amdgcn_readfirstlane(c0[l].x);
            ri0[l] = __builtin_amdgcn_readfirstlane(c0[l].y);
            id0[l] = load_id(a, P, l, ri0[l], cnt0[l], 0);
        }
        for (int n = T - 1; n >= 0; --n) {
            __builtin_amdgcn_s_waitcnt(kWaitVm0);
            int cnt1[NL], ri1[NL], id1[NL];
#pragma unroll
            for (int l = 0; l < NL; ++l) {
                cnt1[l] = __builtin_amdgcn_readfirstlane(c1[l].x);
                ri1[l] = __builtin_amdgcn_readfirstlane(c1[l].y);
                c1[l] = load_cr(P, l, max(n - 2, 0));
                id1[l] = load_id(a, P, l, ri1[l], cnt1[l], 0);
            }
            // ---- adjoint free dynamics, trajectory, adjoint ring
#pragma unroll
            for (int l = 0; l < NL; ++l) {
                const BwdLayer& y = a.ly[l];
                if (j >= y.n) continue;
                if (n <= T - 2) {
                    const double v = lv[l];
                    lI[l] = __dadd_rn(__dmul_rn(a.beta, lI[l]), __dmul_rn(a.cc, v));
                    lv[l] = __dmul_rn(a.alpha, v);
                }
                const double d = __dsub_rn(lI[l], lv[l]);
                P.tr[l][(size_t)n * LT] = make_double2(lI[l], d);
                if (y.ring_lds >= 0) ((lds_f64*)(smem + y.ring_lds))[(n % y.S) * 64 + lane] = d;
            }
            const int rounds = rounds_of(cnt0);
            for (int rd = 0; rd < rounds; ++rd) {
                // this lane's spike among the round's of each layer (position
                // + 1, 0: none), its I- and extra jump numerator
                int mine[NL], off[NL], nr[NL];
                float I[NL];
                double A2[NL];
                int K = 0;
#pragma unroll
                for (int l = 0; l < NL; ++l) {
                    const int q0 = rd * KC;
                    nr[l] = min(max(cnt0[l] - q0, 0), KC);
                    off[l] = K;
                    K += nr[l];
                    const int id = (rd == 0) ? id0[l] : load_id(a, P, l, ri0[l], cnt0[l], q0);
                    pos[l * 64 + lane] = 0;
                    const int o = id - g * 64;
                    if ((int)lane < nr[l] && o >= 0 && o < 64) pos[l * 64 + o] = lane + 1;
                    // other lanes wrote this lane's entry: the read must
                    // not be folded into this lane's own stores (the wave's
                    // LDS accesses are in order)
                    asm volatile("" ::: "memory");
                    mine[l] = pos[l * 64 + lane];
                    I[l] = 0.0f;
                    A2[l] = 0.0;
                    if (mine[l]) {
                        const int rr = ri0[l] + q0 + mine[l] - 1;
                        I[l] = P.recI[l][rr];
                        A2[l] = P.A2[l] ? P.A2[l][rr] : 0.0;
                    }
                }
                lds_barrier();                                   // ring rows in, shares free
                lds_barrier();                                   // shares written
                const bool ok = exchange(a, c, g, rnd++, K, off, nr, rof, nring);
                asm volatile("" ::: "memory");                   // the slot totals of other lanes
                if (!ok) {
                    if (lane == 0) *flag(a) = 1;
                    lds_barrier();                               // the gather waves see the flag
                    return;
                }
#pragma unroll
                for (int l = 0; l < NL; ++l) {
                    if (!mine[l]) continue;
                    const double A = A2[l] + tot[off[l] + mine[l] - 1];
                    // tau_m dV/dt just before the crossing is I- - theta (V- = theta)
                    const double den = __dsub_rn((double)I[l], a.theta);
                    if (den > 0.0)
                        lv[l] = __dadd_rn(lv[l], __dadd_rn(__dmul_rn(a.theta, lv[l]), A) / den);
                    else
                        ++deg;
                }
            }
#pragma unroll
            for (int l = 0; l < NL; ++l) {
                cnt0[l] = cnt1[l];
                ri0[l] = ri1[l];
                id0[l] = id1[l];
            }
        }
        if (deg) atomicAdd(&a.st->degenerate, deg);
    }

    static __device__ void run(const CoreBwdArgs& a) {
        if (a.st->cl_abort) return;
        const int wave = threadIdx.x >> 6;
        int c, g;
        cluster_rank((int)blockIdx.x, a.cl.G, c, g);
        const int b = a.cl.b0 + c;
        if (wave == 0 && (threadIdx.x & 63) == 0) *flag(a) = 0;
        __syncthreads();
        if (wave == 0) {
            neuron_wave(a, b, c, g);
            return;
        }
        int r = 0;
#pragma unroll
        for (int l = 0; l < NL; ++l)
#pragma unroll
            for (int pp = 0; pp < NP; ++pp)
                if (pp < a.ly[l].npost) {
                    if (r == wave - 1) {
                        gather_wave(a, b, g, r, l, pp);
                        return;
                    }
                    ++r;
                }
    }
};

template <int NL, int NP>
__global__ void __launch_bounds__(64 * (1 + NL * NP)) backward_cluster_kernel(CoreBwdArgs a) {
    BwdCluster<NL, NP>::run(a);
}

// ------------------------------------------------------------------ grouping

// One workgroup per sample: counting sort of the sample's spikes by
// presynaptic neuron (LDS histogram, block-wide scan), the steps scattered
// into LDS (or, for a sample with more spikes than the LDS stage holds, into
// device memory), each neuron's steps sorted (thread per neuron, insertion
// sort: the spikes arrive in step order, so a neuron's list is nearly
// sorted), then written out.
__global__ void __launch_bounds__(1024) group_kernel(GroupArgs a) {
    if (a.st->bad_input) return;
    const int b = blockIdx.x, tid = threadIdx.x, nt = blockDim.x;
    const int lane = tid & 63, wv = tid >> 6;
    const int start = a.cnt ? b * a.off_stride : a.off[b];
    const int end = a.cnt ? start + a.cnt[b] : a.end[b + 1];
    const int cnt = end - start;
    int* h = reinterpret_cast<int*>(smem);        // [n + 1] counts, then cursors (segment ends)
    int* wsum = h + a.n + 1;                      // [16] per-wave sums
    unsigned short* stage = reinterpret_cast<unsigned short*>(wsum + 16);   // [stage_cap]
    const bool in_lds = cnt <= a.stage_cap;
    unsigned short* dst = in_lds ? stage : a.g_step + start;
    for (int i = tid; i <= a.n; i += nt) h[i] = 0;
    __syncthreads();
    for (int e = start + tid; e < end; e += nt) atomicAdd(&h[a.neuron[e]], 1);
    __syncthreads();
    // exclusive scan of h[0 .. n): thread tid sums a contiguous segment, the
    // segment sums are scanned within each wave (shuffles) and across waves
    const int seg = (a.n + nt - 1) / nt;
    const int i0 = min(tid * seg, a.n), i1 = min(i0 + seg, a.n);
    int s = 0;
    for (int i = i0; i < i1; ++i) s += h[i];
    int incl = s;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const int y = __shfl_up(incl, d, 64);
        if (lane >= d) incl += y;
    }
    if (lane == 63) wsum[wv] = incl;
    __syncthreads();
    int run = incl - s;
    for (int w = 0; w < wv; ++w) run += wsum[w];
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
        dst[pos] = (unsigned short)a.step[e];
    }
    __syncthreads();
    // h[i] is now the end of neuron i's segment
    for (int i = tid; i < a.n; i += nt) {
        const int lo = i ? h[i - 1] : 0, hi = h[i];
        for (int x = lo + 1; x < hi; ++x) {
            const int v = dst[x];
            int y = x - 1;
            while (y >= lo && dst[y] > v) {
                dst[y + 1] = dst[y];
                --y;
            }
            dst[y + 1] = (unsigned short)v;
        }
    }
    if (!in_lds) return;
    __syncthreads();
    for (int x = tid; x < cnt; x += nt) a.g_step[start + x] = stage[x];
}

// ------------------------------------------------------------------ gradients

// dL/dw_ij = -tau_s sum_spikes lambda_I,j(t + d_ij) and dL/dd_ij = -w_ij
// sum_spikes (lambda_I - lambda_V)_j(t + d_ij), per step of delay (x dt).
//
// Workgroup = (post layer, block of J posts, block of samples).  The J x V
// synapses into the block (V presynaptic neurons over the layer's
// projections) are dealt to lanes: lane l owns pairs p = l + nt k, post
// p % J of presynaptic neuron p / J.  Within a wave the neurons are adjacent
// (similar spike counts, little divergence) and a lane's neurons lie nt / J
// apart, so every lane sums about the same number of spikes however the
// input concentrates on some channels.  Per sample the J post trajectories
// (step-major, [step][post], so the J lanes of a presynaptic neuron read J
// consecutive 16-byte cells of a row, in different banks, plus a zero row)
// and the sample's grouped spike steps are staged in LDS; each lane sums, per
// synapse, in sample then spike order, lambda_I and lambda_I - lambda_V at
// the delayed arrivals in fp64; the weight multiplies the delay sum once at
// the end.  Sample blocks are reduced in a fixed order: no atomics,
// deterministic.
//
// Workgroups come in units of four J-post blocks that share lines of the
// [B][T][N] trajectories; a unit's four blocks have indices 8 apart, so with
// round-robin dispatch over the 8 XCDs they run on one XCD and share its L2.

// n dwords from src to dst in LDS (both 4-byte aligned) as direct loads into
// LDS: wave w of nw takes the 64-dword chunks w, w + nw, ...; the caller
// waits for them (vmcnt) before a barrier.
__device__ inline void lds_dwords(const void* src, void* dst, int n, int w, int nw, int lane) {
    for (int c = w; c * 64 < n; c += nw) {
        const int i = c * 64 + lane;
        if (i < n)
            __builtin_amdgcn_global_load_lds(static_cast<const char*>(src) + (size_t)i * 4,
                                             (lds_ptr_t)(static_cast<char*>(dst) + (size_t)c * 256), 4, 0, 0);
    }
}

// Rows [0, W) of J consecutive posts (row r at src + r ld) into dst [W][J]
// in LDS as direct 16-byte loads: one wave load covers 64 / J rows (lane:
// row lane / J, post lane % J; posts past nj repeat the last one, a cell
// that is never read).
template <int J>
__device__ inline void lds_rows(const double2* src, int ld, int nj, double2* dst, int W, int w, int nw,
                                int lane) {
    constexpr int R = 64 / J;
    const int r = lane / J, q = min(lane % J, nj - 1);
    for (int c = w; c * R < W; c += nw) {
        const int row = c * R + r;
        if (row < W)
            __builtin_amdgcn_global_load_lds(src + (size_t)row * ld + q, (lds_ptr_t)(dst + (size_t)c * 64), 16,
                                             0, 0);
    }
}

template <int J, int KL, bool WIN>
__global__ void __launch_bounds__(1024) gradients_kernel(GradArgs a) {
    const int tid = threadIdx.x, nt = blockDim.x;
    int g = 0;
    while (g + 1 < a.ngroups && (int)blockIdx.x >= a.grp[g + 1].blk0) ++g;
    const GradGroup& G = a.grp[g];
    const int local = (int)blockIdx.x - G.blk0;
    const int unit = (local / 32) * 8 + (local % 8), u = (local % 32) / 8;
    const int LG = (G.jb + 3) / 4;
    if (unit >= LG * a.SB) return;
    const int jb = (unit / a.SB) * 4 + u, sb = unit % a.SB;
    if (jb >= G.jb) return;
    const int nq = G.nq, j0 = jb * J, nj = min(J, nq - j0);
    const int T = a.T;
    const int TW = WIN ? a.TW : a.T;                            // steps per trajectory window
    double2* st = reinterpret_cast<double2*>(smem);            // [TW + 1][J]
    int* gl = reinterpret_cast<int*>(smem + (size_t)J * (TW + 1) * sizeof(double2));   // [glcap]
    unsigned short* sp = reinterpret_cast<unsigned short*>(gl + a.glcap);               // [spcap + 8]
    const int lane = tid & 63, nw = nt >> 6;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const double2* tr = G.out ? a.tr_out : a.tr_lif;
    const int LN = G.out ? a.C : a.lif_total;
    const int n0 = G.npre[0], n1 = (G.np > 1) ? G.npre[1] : 0;
    const int vtot = n0 + n1;
    const int* go0 = a.g_off[G.pre[0]];
    const int* go1 = a.g_off[G.pre[G.np > 1 ? 1 : 0]];
    const unsigned short* gs0 = a.g_step[G.pre[0]];
    const unsigned short* gs1 = a.g_step[G.pre[G.np > 1 ? 1 : 0]];
    const int b0 = sb * a.bs, b1 = min(a.B, b0 + a.bs);
    for (int pbase = 0; pbase < J * vtot; pbase += nt * KL) {
        // this lane's synapses, one word each: presynaptic index (bits 0-15),
        // post within the block (16-19), projection part (20), slot (21-28);
        // -1: none
        int dsc[KL];
#pragma unroll
        for (int k = 0; k < KL; ++k) {
            const int p = pbase + tid + nt * k;
            const int v = p / J, q = p % J;
            dsc[k] = -1;
            if (p < J * vtot && q < nj) {
                const int pi = (v >= n0) ? 1 : 0, i = v - (pi ? n0 : 0);
                const uint2 e = a.ws[a.woff[G.p[pi]] + (size_t)i * nq + j0 + q];
                dsc[k] = i | (q << 16) | (pi << 20) | ((int)e.y << 21);
            }
        }
        double su[KL], sd[KL];
#pragma unroll
        for (int k = 0; k < KL; ++k) {
            su[k] = 0.0;
            sd[k] = 0.0;
        }
        // the list bounds of the first sample (those of the next are loaded
        // while a sample is staged)
        int s0 = go0[(size_t)b0 * (n0 + 1)], e0 = go0[(size_t)b0 * (n0 + 1) + n0];
        int s1 = n1 ? go1[(size_t)b0 * (n1 + 1)] : 0, e1 = n1 ? go1[(size_t)b0 * (n1 + 1) + n1] : 0;
        for (int b = b0; b < b1; ++b) {
            __syncthreads();                                       // the last sample's reads are done
            // (LDS stores first: the compiler waits for the direct loads
            // before any LDS store that follows them)
            if (tid < J) st[min(TW, T) * J + tid] = make_double2(0.0, 0.0);   // row W: no arrival
            // Staging, as direct loads into LDS (no registers, all in flight
            // at once, one memory round trip per sample): the spike-list
            // offsets of both presynaptic layers, the grouped spike steps
            // (16-bit, copied as aligned dwords: list 0 from s0 rounded down
            // to even, list 1 from an even LDS index), the first window of the
            // J post trajectories.
            const int a0 = s0 & ~1, a1 = s1 & ~1;
            const int L0 = e0 - a0, A1 = (L0 + 1) & ~1, L1 = n1 ? e1 - a1 : 0;
            const bool in_lds = A1 + L1 + 1 <= a.spcap;
            const int off0 = -a0, off1 = A1 - a1;                 // LDS index = x + off
            if (b + 1 < b1) {                                      // the next sample's bounds
                const size_t o0 = (size_t)(b + 1) * (n0 + 1), o1 = (size_t)(b + 1) * (n1 + 1);
                s0 = go0[o0];
                e0 = go0[o0 + n0];
                s1 = n1 ? go1[o1] : 0;
                e1 = n1 ? go1[o1 + n1] : 0;
            }
            lds_dwords(go0 + (size_t)b * (n0 + 1), gl, n0 + 1, wv, nw, lane);
            if (n1) lds_dwords(go1 + (size_t)b * (n1 + 1), gl + n0 + 1, n1 + 1, wv, nw, lane);
            if (in_lds) {
                lds_dwords(gs0 + a0, sp, (L0 + 1) >> 1, wv, nw, lane);
                if (L1 > 0) lds_dwords(gs1 + a1, sp + A1, (L1 + 1) >> 1, wv, nw, lane);
            }
            const size_t base = (size_t)b * T * LN + G.off + j0;
            lds_rows<J>(tr + base, LN, nj, st, min(TW, T), wv, nw, lane);
            __builtin_amdgcn_s_waitcnt(0);
            __syncthreads();
            // spike lists of this lane's neurons (offsets into g_step)
            int lo[KL], hi[KL];
#pragma unroll
            for (int k = 0; k < KL; ++k) {
                const int i = dsc[k] & 0xFFFF, pi = (dsc[k] >> 20) & 1;
                const int* go = gl + (pi ? n0 + 1 : 0);
                lo[k] = (dsc[k] >= 0) ? go[i] : 0;
                hi[k] = (dsc[k] >= 0) ? go[i + 1] : 0;
            }
            // the J post trajectories of the sample, in windows of TW steps
            // (one window unless the trial is long); a synapse's spikes are
            // taken in step order, window by window, from a cursor
            for (int w0 = 0; w0 < T; w0 += TW) {
                const int W = min(TW, T - w0), wend = w0 + W;
                if (w0 > 0) {
                    __syncthreads();                                // the last window's reads are done
                    if (tid < J) st[W * J + tid] = make_double2(0.0, 0.0);
                    lds_rows<J>(tr + base + (size_t)w0 * LN, LN, nj, st, W, wv, nw, lane);
                    __builtin_amdgcn_s_waitcnt(0);
                    __syncthreads();
                }
#pragma unroll
                for (int k = 0; k < KL; ++k) {
                    // the descriptor is made opaque here, so that what derives
                    // from it is recomputed per sample instead of being hoisted
                    // out of the sample loop (KL sets of it do not fit in
                    // registers beside the sums: the spills cost HBM writes)
                    int dk = dsc[k];
                    asm volatile("" : "+v"(dk));
                    if (dk < 0) continue;
                    const int pi = (dk >> 20) & 1, sl = (dk >> 21) & 0xFF;
                    const double2* stk = st + ((dk >> 16) & 0xF);            // row: arrival - w0
                    const unsigned short* gs = pi ? gs1 : gs0;
                    const int off = pi ? off1 : off0;
                    double pu = su[k], pd = sd[k];
                    // four spikes at a time: their reads issued together, their
                    // terms added in spike order; the arrivals ascend, so the
                    // window's spikes are a prefix from the cursor.  The loop
                    // comes in two copies, spike steps in LDS or in device
                    // memory (one choice per sample), and a term past the
                    // window or past the list reads the zero row W and adds +0
                    // (the sums start at +0, so they never hold -0 and +0
                    // changes nothing): no branch and no select inside.
                    int x = lo[k];
                    const int h = hi[k];
                    auto spikes = [&](auto in_lds_tag) {
                        constexpr bool SPL = decltype(in_lds_tag)::value;
                        for (; x < h; x += 4) {
                            // the four reads unconditional and issued together
                            // (the empty asm keeps the compiler from moving each
                            // behind its own branch and wait)
                            int t[4], m[4];
#pragma unroll
                            for (int u = 0; u < 4; ++u) {
                                // (the LDS list has slack past its end:
                                // no clamp there)
                                t[u] = SPL ? (int)sp[x + u + off] : gs[min(x + u, h - 1)];
                            }
                            asm volatile("" : "+v"(t[0]), "+v"(t[1]), "+v"(t[2]), "+v"(t[3]));
#pragma unroll
                            for (int u = 0; u < 4; ++u) m[u] = (x + u < h) ? t[u] + sl : T;   // T: no arrival
                            double2 ud[4];
#pragma unroll
                            for (int u = 0; u < 4; ++u) ud[u] = stk[min((unsigned)(m[u] - w0), (unsigned)W) * J];
#pragma unroll
                            for (int u = 0; u < 4; ++u) {
                                pu = __dadd_rn(pu, ud[u].x);
                                pd = __dadd_rn(pd, ud[u].y);
                            }
                            if constexpr (WIN) {
                                if (m[3] >= wend) {
                                    x += (m[0] < wend) + (m[1] < wend) + (m[2] < wend);
                                    break;
                                }
                            }
                        }
                    };
                    if (in_lds)
                        spikes(std::true_type{});
                    else
                        spikes(std::false_type{});
                    if constexpr (WIN) lo[k] = min(x, h);
                    su[k] = pu;
                    sd[k] = pd;
                }
            }
        }
#pragma unroll
        for (int k = 0; k < KL; ++k) {
            if (dsc[k] < 0) continue;
            const int p = G.p[(dsc[k] >> 20) & 1];
            const size_t kk = (size_t)(dsc[k] & 0xFFFF) * nq + j0 + ((dsc[k] >> 16) & 0xF);
            if (a.SB == 1) {
                const double w = (double)__uint_as_float(a.ws[a.woff[p] + kk].x);
                a.dW[p][kk] = (float)(-(double)a.tau_s * su[k]);
                a.dD[p][kk] = (float)(-(double)a.dt * (w * sd[k]));
            } else {
                const size_t gi = (size_t)a.woff[p] + kk;
                a.part[((size_t)sb * 2 + 0) * a.nparams + gi] = su[k];
                a.part[((size_t)sb * 2 + 1) * a.nparams + gi] = sd[k];
            }
        }
    }
}

// Extra jump numerator of every record of a LIF layer: dst = base + dlp +
// nterm[neuron of the record] (each may be absent), for the stored records of
// each sample.
__global__ void add_lp_kernel(double* dst, const double* base, const float* dlp, const double* nterm,
                              const int* rec_n, const int* cnt, int B, int cap) {
    const int b = blockIdx.y;
    const int r = blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= B || r >= min(cnt[b], cap)) return;
    const size_t k = (size_t)b * cap + r;
    double v = base ? base[k] : 0.0;
    if (dlp) v += (double)dlp[k];
    if (nterm) v += nterm[rec_n[k]];
    dst[k] = v;
}

// Sample-block partial sums, added in block order.
__global__ void grad_reduce_kernel(GradArgs a, int P) {
    const long long g = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (g >= a.nparams) return;
    int p = 0;
    while (p + 1 < P && g >= a.woff[p + 1]) ++p;
    double su = 0.0, sd = 0.0;
    for (int sb = 0; sb < a.SB; ++sb) {
        su += a.part[((size_t)sb * 2 + 0) * a.nparams + g];
        sd += a.part[((size_t)sb * 2 + 1) * a.nparams + g];
    }
    const long long kk = g - a.woff[p];
    const double w = (double)__uint_as_float(a.ws[g].x);
    a.dW[p][kk] = (float)(-(double)a.tau_s * su);
    a.dD[p][kk] = (float)(-(double)a.dt * (w * sd));
}

}  // namespace

// ------------------------------------------------------------------ launchers

hipError_t launch_readout_adjoint(const ReadoutBwdArgs& a, int threads, size_t lds, hipStream_t s) {
    hipLaunchKernelGGL(readout_adjoint_kernel, dim3(a.B), dim3(threads), lds, s, a);
    return hipGetLastError();
}

template <int MAXT, int NL, int NP>
static void launch_core3(const CoreBwdArgs& a, bool rl, int threads, size_t lds, hipStream_t s) {
    constexpr int KP = bwd_prefetch(NL);
    if (rl)
        hipLaunchKernelGGL((backward_core_kernel<MAXT, NL, KP, NP, true>), dim3(a.B), dim3(threads),
                           lds, s, a);
    else
        hipLaunchKernelGGL((backward_core_kernel<MAXT, NL, KP, NP, false>), dim3(a.B), dim3(threads),
                           lds, s, a);
}

template <int MAXT>
static bool launch_core_t(const CoreBwdArgs& a, int n_lif, int np, bool rl, int threads, size_t lds,
                          hipStream_t s) {
    switch (n_lif * 4 + np) {
        case 4 + 0: launch_core3<MAXT, 1, 0>(a, rl, threads, lds, s); return true;
        case 4 + 1: launch_core3<MAXT, 1, 1>(a, rl, threads, lds, s); return true;
        case 8 + 1: launch_core3<MAXT, 2, 1>(a, rl, threads, lds, s); return true;
        case 8 + 2: launch_core3<MAXT, 2, 2>(a, rl, threads, lds, s); return true;
        case 12 + 1: launch_core3<MAXT, 3, 1>(a, rl, threads, lds, s); return true;
        case 12 + 2: launch_core3<MAXT, 3, 2>(a, rl, threads, lds, s); return true;
        case 16 + 1: launch_core3<MAXT, 4, 1>(a, rl, threads, lds, s); return true;
        case 16 + 2: launch_core3<MAXT, 4, 2>(a, rl, threads, lds, s); return true;
        default: return false;
    }
}

hipError_t launch_backward_core(const CoreBwdArgs& a, int n_lif, int threads, size_t lds,
                                hipStream_t s) {
    if (n_lif < 1 || n_lif > SNN_MAX_LIF || threads != 64 * a.NW) return hipErrorInvalidValue;
    int np = 0;
    bool rl = true;
    for (int l = 0; l < n_lif; ++l) {
        np = max(np, a.ly[l].npost);
        if (a.ly[l].ring_lds == -1) rl = false;
        for (int pp = 0; pp < a.ly[l].npost; ++pp)
            if (a.ly[l].qring_lds[pp] < 0) rl = false;
    }
    const bool ok = (threads <= 256) ? launch_core_t<256>(a, n_lif, np, rl, threads, lds, s)
                                     : launch_core_t<1024>(a, n_lif, np, rl, threads, lds, s);
    if (!ok) return hipErrorInvalidValue;
    return hipGetLastError();
}

// Cluster mode: a neuron wave and one gather wave per LIF -> LIF
// projection per workgroup, G workgroups per sample, one cooperative launch
// (the runtime refuses a grid that cannot be resident at once, so every wait
// of a cluster ends).
template <int NL, int NP>
static const void* bcl_fn() {
    return (const void*)backward_cluster_kernel<NL, NP>;
}

static const void* bcl_kernel(int n_lif, int np) {
    switch (n_lif * 4 + np) {
        case 4 + 1: return bcl_fn<1, 1>();
        case 8 + 1: return bcl_fn<2, 1>();
        case 8 + 2: return bcl_fn<2, 2>();
        case 12 + 1: return bcl_fn<3, 1>();
        case 12 + 2: return bcl_fn<3, 2>();
        case 16 + 1: return bcl_fn<4, 1>();
        case 16 + 2: return bcl_fn<4, 2>();
        default: return nullptr;
    }
}

hipError_t launch_backward_core_cluster(const CoreBwdArgs& a, int n_lif, int np, int grid, int threads,
                                        size_t lds, hipStream_t s) {
    const void* f = bcl_kernel(n_lif, np);
    int rings = 0;
    for (int l = 0; l < n_lif; ++l) rings += a.ly[l].npost;
    if (!f || a.cl.G < 1 || grid < a.cl.G || grid % a.cl.G || threads != 64 * (1 + rings) ||
        rings > n_lif * np)
        return hipErrorInvalidValue;
    CoreBwdArgs arg = a;
    void* args[] = {&arg};
    return hipLaunchCooperativeKernel(f, dim3(grid), dim3(threads), args, (unsigned)lds, s);
}

hipError_t backward_cluster_occupancy(int n_lif, int np, int threads, size_t lds, int* blocks_per_cu) {
    const void* f = bcl_kernel(n_lif, np);
    if (!f) return hipErrorInvalidValue;
    return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks_per_cu, f, threads, lds);
}

hipError_t launch_group(const GroupArgs& a, int B, hipStream_t s) {
    if (a.stage_cap < 0) return hipErrorInvalidValue;
    const size_t lds = sizeof(int) * ((size_t)a.n + 1 + 16) + sizeof(unsigned short) * (size_t)a.stage_cap;
    hipLaunchKernelGGL(group_kernel, dim3(B), dim3(1024), lds, s, a);
    return hipGetLastError();
}

hipError_t launch_gradients(const GradArgs& a, int J, int KL, int threads, size_t lds, hipStream_t s) {
    const bool win = a.TW < a.T;
#define SNN_GRAD(JJ, KK, WW)                                                                         \
    if (J == JJ && KL == KK && win == WW) {                                                          \
        hipLaunchKernelGGL((gradients_kernel<JJ, KK, WW>), dim3(a.nblk), dim3(threads), lds, s, a); \
        return hipGetLastError();                                                                    \
    }
    SNN_GRAD(8, 4, false)
    SNN_GRAD(8, 8, false)
    SNN_GRAD(4, 4, false)
    SNN_GRAD(4, 8, false)
    SNN_GRAD(2, 4, false)
    SNN_GRAD(2, 8, false)
    SNN_GRAD(1, 4, false)
    SNN_GRAD(1, 8, false)
    SNN_GRAD(8, 4, true)
    SNN_GRAD(8, 8, true)
#undef SNN_GRAD
    return hipErrorInvalidValue;
}

hipError_t launch_add_lp(double* dst, const double* base, const float* dlp, const double* nterm,
                         const int* rec_n, const int* cnt, int B, int cap, hipStream_t s) {
    if (B <= 0 || cap <= 0) return hipSuccess;
    hipLaunchKernelGGL(add_lp_kernel, dim3(grid_for(cap, 256), B), dim3(256), 0, s, dst, base, dlp,
                       nterm, rec_n, cnt, B, cap);
    return hipGetLastError();
}

hipError_t launch_grad_reduce(const GradArgs& a, int P, hipStream_t s) {
    hipLaunchKernelGGL(grad_reduce_kernel, dim3(grid_for(a.nparams, 256)), dim3(256), 0, s, a, P);
    return hipGetLastError();
}

#define CORE_FNS2(M, R)                                                                          \
    (const void*)backward_core_kernel<M, 1, bwd_prefetch(1), 0, R>, (const void*)backward_core_kernel<M, 1, bwd_prefetch(1), 1, R>, \
    (const void*)backward_core_kernel<M, 2, 4, 1, R>, (const void*)backward_core_kernel<M, 2, 4, 2, R>, \
    (const void*)backward_core_kernel<M, 3, 4, 1, R>, (const void*)backward_core_kernel<M, 3, 4, 2, R>, \
    (const void*)backward_core_kernel<M, 4, 4, 1, R>, (const void*)backward_core_kernel<M, 4, 4, 2, R>
#define CORE_FNS(M) CORE_FNS2(M, true), CORE_FNS2(M, false)
#define CORE_FNS_CL                                                                               \
    bcl_fn<1, 1>(), bcl_fn<2, 1>(), bcl_fn<2, 2>(), bcl_fn<3, 1>(), bcl_fn<3, 2>(), bcl_fn<4, 1>(),   \
        bcl_fn<4, 2>()

hipError_t set_backward_lds_limits(size_t bytes, int* bad) {
    const void* fns[] = {(const void*)readout_adjoint_kernel, CORE_FNS(256), CORE_FNS(1024),
                         (const void*)group_kernel, (const void*)gradients_kernel<8, 4, false>,
                         (const void*)gradients_kernel<8, 8, false>, (const void*)gradients_kernel<4, 4, false>,
                         (const void*)gradients_kernel<4, 8, false>, (const void*)gradients_kernel<2, 4, false>,
                         (const void*)gradients_kernel<2, 8, false>, (const void*)gradients_kernel<1, 4, false>,
                         (const void*)gradients_kernel<1, 8, false>, (const void*)gradients_kernel<8, 4, true>,
                         (const void*)gradients_kernel<8, 8, true>, CORE_FNS_CL};
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
