/*
 * snn_oracle.c -- plain single-threaded CPU oracle for grid EventProp with
 * learnable synaptic delays (Mészáros, Knight, Nowotny, arXiv 2501.07331).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the checker, not the product: only
 * the tests, the smoke check and the bench's CPU-baseline leg may load it.  It
 * shares no code, header, table or constant generator with the HIP library.
 *
 * What it computes (per sample; samples are independent):
 *
 *   Forward, n = 0 .. T-1, state V = I = 0 at t = 0, one delay ring
 *   R_p[S][N_post] = 0 per projection p, S = max_delay + 1 (at least the
 *   projection's largest delay + 1; the ring depth does not change results):
 *     1. every non-input neuron: V- = fma(alpha, V, gamma*I), I- = beta*I
 *        (n = 0: V- = I- = 0).  alpha = e^{-dt/tau_m}, beta = e^{-dt/tau_s},
 *        gamma = tau_s/(tau_s - tau_m) (beta - alpha): the exact solution of
 *        the free dynamics of Table 1 (tau_m V' = -V + I, tau_s I' = -I) over
 *        one step.
 *     2. LIF neurons: spike if V- >= theta, record (n, i, I-), reset V = 0
 *        (Table 1 transition condition and jump).  LI neurons: V = V-.
 *     3. emit: projections in order, presynaptic spikes at n in ascending
 *        index, posts ascending: m = n + slot_ij; if m <= T-1,
 *        R_p[m mod S][j] += w_ij (the delayed current jump of Table 1).
 *     4. arrive: I = I- + R_p[n mod S][j] for the projections p into the
 *        layer, in projection order; those cells are cleared.
 *     5. readout of the LI layer: sum  acc_k += V_k;  max  first argmax.
 *   z_k = s * acc_k (sum) or max_n V_k (max); CE loss; g = dL/dz.
 *   With the spike-time loss (OR_LOSS_DMSE) the last layer is LIF instead:
 *   z_k is the first spike time of output neuron k in ms (n dt; T dt when
 *   it never fires) and the loss is the time-invariant MSE of the Methods,
 *   L_b = 1/2 sum_{i != c} (t_i - t_c - Delta)^2 with c the label.
 *
 *   Backward, n = T-1 .. 0, lambda = 0, trajectory H[n][j] of (lambda_V,
 *   lambda_I):
 *     1. n <= T-2: lambda_I <- beta lambda_I + c lambda_V, lambda_V <- alpha
 *        lambda_V (exact one-step solution of the adjoint ODEs of Table 1,
 *        c = tau_m/(tau_m - tau_s) (alpha - beta)).
 *     2. H[n][j] = (lambda_V, lambda_I): the "+" values at n.
 *     3. LI loss source: sum  lambda_V -= s g_k / tau_m every step;
 *        max  lambda_V -= g_k / tau_m at the first argmax step.
 *     4. every LIF spike (n, i, I-): with (v, u) = H[m][j] at the arrival
 *        m = n + slot_ij <= T-1 of each post j, A_i = sum_j w_ij (v - u);
 *        tau_m V-dot^- = I- - theta at a crossing, so
 *        lambda_V <- lambda_V + (theta lambda_V + A_i) / (I- - theta)
 *        (the lambda_V jump of Table 1 with the delayed postsynaptic sum);
 *        skipped and counted as degenerate if I- - theta <= 0.  A
 *        spike-time loss l_p adds its derivative dl_p/dt_k to the numerator
 *        (Table 1 backward transition; Methods, time-invariant MSE): given
 *        per record in rec_dlp.  There is no LI source then.
 *   Then the gradient sums over every presynaptic spike (n, i) (inputs and
 *   LIF records), in spike order, and post j with m = n + slot <= T-1:
 *     SU_ij += u,  SD_ij += w_ij (u - v),   (v, u) = H[m][j];
 *   dL/dw = -tau_s SU and dL/dd = -dt SD per step of delay: the weight and
 *   delay gradients of Table 1 / the Methods, with the post adjoints taken at
 *   the delayed arrival time.
 *
 * mode 0 runs the backward in fp64 with fp64 constants: the definition the
 * parity tests judge against.
 * mode 1 rounds every backward operation to fp32, in the order written above
 * (the batch sums SU, SD and the jump's postsynaptic sum A included): how far
 * an fp32 evaluation of the same expressions lands from the fp64 one, a noise
 * floor reported beside the parity results.
 * The forward is fp32 with no contraction in both modes: spike decisions are
 * taken in fp32, the precision of the forward pass.
 *
 * Delays: slot = rint(D) (half to even) clamped to [0, pmax[p]] per
 * projection p (pmax NULL: max_delay for every projection), NaN -> 0.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define OR_INPUT 0
#define OR_LIF 1
#define OR_LI 2
#define OR_LOSS_CE_SUM 0
#define OR_LOSS_CE_MAX 1
#define OR_LOSS_DMSE 2

#define OR_OK 0
#define OR_EINVAL (-1)
#define OR_ENOMEM (-2)
#define OR_EOVERFLOW (-4)

#define OR_MAXL 16
#define OR_MAXP 32

typedef struct {
    int L;
    int n[OR_MAXL], kind[OR_MAXL], rec[OR_MAXL];
    int P;
    int pre[OR_MAXP], post[OR_MAXP];
    long w_off[OR_MAXP];
    long n_params;
    int st_off[OR_MAXL];    /* offset of layer l in the flat non-input state */
    int n_state;
    int lif_idx[OR_MAXL];   /* index among LIF layers, -1 otherwise */
    int n_lif;
} topo_t;

static int build_topo(topo_t* t, int L, const int* n, const int* kind, const int* rec) {
    if (L < 2 || L > OR_MAXL) return OR_EINVAL;
    memset(t, 0, sizeof(*t));
    t->L = L;
    for (int l = 0; l < L; ++l) {
        t->n[l] = n[l];
        t->kind[l] = kind[l];
        t->rec[l] = rec[l];
        if (n[l] <= 0) return OR_EINVAL;
        if (l == 0 && kind[l] != OR_INPUT) return OR_EINVAL;
        if (l > 0 && l < L - 1 && kind[l] != OR_LIF) return OR_EINVAL;
        if (l == L - 1 && kind[l] != OR_LI && kind[l] != OR_LIF) return OR_EINVAL;
        if (rec[l] && kind[l] != OR_LIF) return OR_EINVAL;
    }
    t->P = 0;
    long off = 0;
    for (int l = 1; l < L; ++l) {
        for (int r = 0; r < 1 + (rec[l] ? 1 : 0); ++r) {
            if (t->P >= OR_MAXP) return OR_EINVAL;
            int p = t->P++;
            t->pre[p] = r ? l : l - 1;
            t->post[p] = l;
            t->w_off[p] = off;
            off += (long)n[t->pre[p]] * n[l];
        }
    }
    t->n_params = off;
    int so = 0, li = 0;
    for (int l = 0; l < L; ++l) {
        t->st_off[l] = so;
        if (l > 0) so += n[l];
        t->lif_idx[l] = (kind[l] == OR_LIF) ? li++ : -1;
    }
    t->n_state = so;
    t->n_lif = li;
    return OR_OK;
}

/* Delay rounding: round half to even, clamp to [0, max_delay]; NaN -> 0.
 * Delays are integer multiples of the time step (Discussion). */
static int delay_slot(float d, int max_delay, long* clamped) {
    float r = rintf(d);
    if (isnan(r) || r < 0.0f) { ++*clamped; return 0; }
    if (r > (float)max_delay) { ++*clamped; return max_delay; }
    return (int)r;
}

/* Slots of every synapse, projection by projection (pmax: largest delay per
 * projection, or NULL for max_delay everywhere); returns OR_EINVAL if a
 * pmax entry lies outside [0, max_delay]. */
static int fill_slots(const topo_t* t, const float* D, int max_delay, const int* pmax,
                      unsigned char* slot, long* clamped) {
    for (int p = 0; p < t->P; ++p) {
        const int dm = pmax ? pmax[p] : max_delay;
        if (dm < 0 || dm > max_delay) return OR_EINVAL;
        const long n_p = (long)t->n[t->pre[p]] * t->n[t->post[p]];
        for (long k = 0; k < n_p; ++k)
            slot[t->w_off[p] + k] = (unsigned char)delay_slot(D[t->w_off[p] + k], dm, clamped);
    }
    return OR_OK;
}

int oracle_constants(float tau_m, float tau_s, float dt, float* out4) {
    if (!(dt > 0.0f) || !(tau_m > 0.0f) || !(tau_s > 0.0f) || tau_m == tau_s) return OR_EINVAL;
    double a = exp(-(double)dt / (double)tau_m);
    double b = exp(-(double)dt / (double)tau_s);
    double g = (double)tau_s / ((double)tau_s - (double)tau_m) * (b - a);
    double c = (double)tau_m / ((double)tau_m - (double)tau_s) * (a - b);
    out4[0] = (float)a;
    out4[1] = (float)b;
    out4[2] = (float)g;
    out4[3] = (float)c;
    return OR_OK;
}

static int check_inputs(const topo_t* t, int B, int T, const int* in_off, const int* in_step,
                        const int* in_neuron) {
    if (B < 0 || T <= 0) return OR_EINVAL;
    if (in_off[0] != 0) return OR_EINVAL;
    for (int b = 0; b < B; ++b) {
        if (in_off[b + 1] < in_off[b]) return OR_EINVAL;
        for (int e = in_off[b]; e < in_off[b + 1]; ++e) {
            if (in_step[e] < 0 || in_step[e] >= T) return OR_EINVAL;
            if (in_neuron[e] < 0 || in_neuron[e] >= t->n[0]) return OR_EINVAL;
            if (e > in_off[b]) {
                long k0 = (long)in_step[e - 1] * t->n[0] + in_neuron[e - 1];
                long k1 = (long)in_step[e] * t->n[0] + in_neuron[e];
                if (k1 <= k0) return OR_EINVAL;   /* sorted by (step, neuron), unique */
            }
        }
    }
    return OR_OK;
}

/*
 * Records are laid out [n_lif][B][cap].  V_trace, if not NULL, receives V- of
 * every non-input neuron at every step, [B][T][n_state].  stats[0] = number of
 * clamped delays.  Returns OR_EOVERFLOW (after a complete forward) if a sample
 * produced more than cap spikes in some layer; counts are still exact.
 */
int oracle_forward(int L, const int* n, const int* kind, const int* rec,
                   float tau_m, float tau_s, float theta, float dt, int max_delay, const int* pmax,
                   int B, int T, int loss, float readout_scale,
                   const int* in_off, const int* in_step, const int* in_neuron,
                   const float* W, const float* D, int cap,
                   int* rec_count, int* rec_step, int* rec_neuron, float* rec_I,
                   float* z, int* nstar, float* V_final, float* I_final,
                   float* V_trace, long* stats) {
    topo_t t;
    int rc = build_topo(&t, L, n, kind, rec);
    if (rc) return rc;
    if (max_delay < 0 || max_delay > 255 || cap < 0) return OR_EINVAL;
    if (loss != OR_LOSS_CE_SUM && loss != OR_LOSS_CE_MAX && loss != OR_LOSS_DMSE) return OR_EINVAL;
    if ((loss == OR_LOSS_DMSE) != (t.kind[L - 1] == OR_LIF)) return OR_EINVAL;
    rc = check_inputs(&t, B, T, in_off, in_step, in_neuron);
    if (rc) return rc;
    float k4[4];
    rc = oracle_constants(tau_m, tau_s, dt, k4);
    if (rc) return rc;
    const float alpha = k4[0], beta = k4[1], gamma = k4[2];
    const int S = max_delay + 1;
    const int C = t.n[L - 1];
    const int out_l = L - 1;

    long clamped = 0;
    unsigned char* slot = (unsigned char*)malloc((size_t)t.n_params);
    float* V = (float*)malloc(sizeof(float) * t.n_state);
    float* I = (float*)malloc(sizeof(float) * t.n_state);
    /* one ring per projection: ring_off[p] columns into a row of ring_w */
    int ring_off[OR_MAXP + 1], ring_w = 0;
    for (int p = 0; p < t.P; ++p) {
        ring_off[p] = ring_w;
        ring_w += t.n[t.post[p]];
    }
    float* ring = (float*)malloc(sizeof(float) * (size_t)S * (ring_w > 0 ? ring_w : 1));
    int* spk = (int*)malloc(sizeof(int) * t.n_state);      /* spikes of this step, per layer */
    int spk_n[OR_MAXL];
    float* acc = (float*)malloc(sizeof(float) * C);
    float* best = (float*)malloc(sizeof(float) * C);
    int* first = (int*)malloc(sizeof(int) * C);
    if (!slot || !V || !I || !ring || !spk || !acc || !best || !first) {
        free(slot); free(V); free(I); free(ring); free(spk); free(acc); free(best); free(first);
        return OR_ENOMEM;
    }
    if (fill_slots(&t, D, max_delay, pmax, slot, &clamped)) {
        free(slot); free(V); free(I); free(ring); free(spk); free(acc); free(best); free(first);
        return OR_EINVAL;
    }

    int overflow = 0;
    for (int b = 0; b < B; ++b) {
        memset(V, 0, sizeof(float) * t.n_state);
        memset(I, 0, sizeof(float) * t.n_state);
        memset(ring, 0, sizeof(float) * (size_t)S * ring_w);
        for (int l = 0; l < L; ++l)
            if (t.lif_idx[l] >= 0) rec_count[(size_t)t.lif_idx[l] * B + b] = 0;
        for (int k = 0; k < C; ++k) first[k] = -1;
        int cur = in_off[b];
        const int end = in_off[b + 1];
        for (int n_ = 0; n_ < T; ++n_) {
            /* 1-2. free dynamics over one step, threshold, reset, record */
            for (int l = 1; l < L; ++l) {
                spk_n[l] = 0;
                for (int j = 0; j < t.n[l]; ++j) {
                    const int s = t.st_off[l] + j;
                    float Vm = 0.0f, Im = 0.0f;
                    if (n_ >= 1) {
                        float gi = gamma * I[s];
                        Vm = fmaf(alpha, V[s], gi);
                        Im = beta * I[s];
                    }
                    if (V_trace) V_trace[((size_t)b * T + n_) * t.n_state + s] = Vm;
                    I[s] = Im;
                    if (t.kind[l] == OR_LIF && Vm >= theta) {
                        V[s] = 0.0f;
                        spk[t.st_off[l] + spk_n[l]++] = j;
                        const int li = t.lif_idx[l];
                        int* cnt = &rec_count[(size_t)li * B + b];
                        if (*cnt < cap) {
                            size_t r = ((size_t)li * B + b) * cap + *cnt;
                            rec_step[r] = n_;
                            rec_neuron[r] = j;
                            rec_I[r] = Im;
                        } else {
                            overflow = 1;
                        }
                        ++*cnt;
                    } else {
                        V[s] = Vm;
                    }
                }
            }
            /* 3. emit into the delay rings */
            int in_lo = cur, in_hi = cur;
            while (in_hi < end && in_step[in_hi] == n_) ++in_hi;
            cur = in_hi;
            for (int p = 0; p < t.P; ++p) {
                const int a = t.pre[p], q = t.post[p];
                const int nq = t.n[q];
                const int cnt = (a == 0) ? in_hi - in_lo : spk_n[a];
                for (int k = 0; k < cnt; ++k) {
                    const int i = (a == 0) ? in_neuron[in_lo + k] : spk[t.st_off[a] + k];
                    const float* wrow = W + t.w_off[p] + (long)i * nq;
                    const unsigned char* srow = slot + t.w_off[p] + (long)i * nq;
                    for (int j = 0; j < nq; ++j) {
                        const int m = n_ + srow[j];
                        if (m <= T - 1) ring[(size_t)(m % S) * ring_w + ring_off[p] + j] += wrow[j];
                    }
                }
            }
            /* 4. arrivals, projection by projection */
            float* row = ring + (size_t)(n_ % S) * ring_w;
            for (int p = 0; p < t.P; ++p) {
                const int q = t.post[p];
                for (int j = 0; j < t.n[q]; ++j) {
                    float* cell = row + ring_off[p] + j;
                    I[t.st_off[q] + j] = I[t.st_off[q] + j] + *cell;
                    *cell = 0.0f;
                }
            }
            /* 5. readout: first spikes of a LIF output layer, or the LI voltages */
            if (loss == OR_LOSS_DMSE) {
                for (int q = 0; q < spk_n[out_l]; ++q) {
                    const int k = spk[t.st_off[out_l] + q];
                    if (first[k] < 0) first[k] = n_;
                }
                continue;
            }
            for (int k = 0; k < C; ++k) {
                const float v = V[t.st_off[out_l] + k];
                if (loss == OR_LOSS_CE_SUM) {
                    acc[k] = (n_ == 0) ? v : acc[k] + v;
                } else if (n_ == 0 || v > best[k]) {
                    best[k] = v;
                    nstar[(size_t)b * C + k] = n_;
                }
            }
        }
        if (loss == OR_LOSS_DMSE) {
            /* first spike times in ms, T dt for a neuron that never fires */
            for (int k = 0; k < C; ++k) {
                const int n0 = first[k] >= 0 ? first[k] : T;
                z[(size_t)b * C + k] = (float)((double)n0 * (double)dt);
                nstar[(size_t)b * C + k] = first[k];
            }
        } else {
            for (int k = 0; k < C; ++k)
                z[(size_t)b * C + k] = (loss == OR_LOSS_CE_SUM) ? readout_scale * acc[k] : best[k];
            if (loss == OR_LOSS_CE_SUM)
                for (int k = 0; k < C; ++k) nstar[(size_t)b * C + k] = -1;
        }
        if (V_final) memcpy(V_final + (size_t)b * t.n_state, V, sizeof(float) * t.n_state);
        if (I_final) memcpy(I_final + (size_t)b * t.n_state, I, sizeof(float) * t.n_state);
    }
    if (stats) stats[0] = clamped;
    free(slot); free(V); free(I); free(ring); free(spk); free(acc); free(best); free(first);
    return overflow ? OR_EOVERFLOW : OR_OK;
}

/* Softmax cross-entropy on z, in fp64.  loss_out[b] = CE_b, loss_out[B] = mean;
 * g[b][k] = (softmax(z_b)_k - [k = y_b]) / B. */
int oracle_loss(int B, int C, const float* z, const int* labels, float* loss_out, float* g) {
    if (B <= 0 || C <= 0) return OR_EINVAL;
    double total = 0.0;
    for (int b = 0; b < B; ++b) {
        const float* zb = z + (size_t)b * C;
        if (labels[b] < 0 || labels[b] >= C) return OR_EINVAL;
        double mx = zb[0];
        for (int k = 1; k < C; ++k) if (zb[k] > mx) mx = zb[k];
        double se = 0.0;
        for (int k = 0; k < C; ++k) se += exp((double)zb[k] - mx);
        const double lse = mx + log(se);
        const double ce = lse - (double)zb[labels[b]];
        loss_out[b] = (float)ce;
        total += ce;
        for (int k = 0; k < C; ++k) {
            double p = exp((double)zb[k] - lse);
            g[(size_t)b * C + k] = (float)((p - (k == labels[b] ? 1.0 : 0.0)) / (double)B);
        }
    }
    loss_out[B] = (float)(total / (double)B);
    return OR_OK;
}

/* Time-invariant MSE on first output spike times (Methods): t_k = z[b][k]
 * in ms, c = labels[b]; L_b = 1/2 sum_{i != c} (t_i - t_c - delta)^2 in
 * fp64; loss_out[b] = L_b, loss_out[B] = mean; dl[b][k] = dL/dt_k of the
 * batch mean: (t_k - t_c - delta)/B for k != c and -sum_{i != c} (t_i - t_c
 * - delta)/B for k = c. */
int oracle_loss_dmse(int B, int C, const float* z, const int* labels, float delta, float* loss_out,
                     double* dl) {
    if (B <= 0 || C <= 0) return OR_EINVAL;
    double total = 0.0;
    for (int b = 0; b < B; ++b) {
        const int c = labels[b];
        if (c < 0 || c >= C) return OR_EINVAL;
        const float* tb = z + (size_t)b * C;
        double L = 0.0, sc = 0.0;
        for (int k = 0; k < C; ++k) {
            if (k == c) continue;
            const double e = (double)tb[k] - (double)tb[c] - (double)delta;
            L += 0.5 * e * e;
            sc += e;
            dl[(size_t)b * C + k] = e / (double)B;
        }
        dl[(size_t)b * C + c] = -sc / (double)B;
        loss_out[b] = (float)L;
        total += L;
    }
    loss_out[B] = (float)(total / (double)B);
    return OR_OK;
}

/* fp32 rounding of a double that holds the exact result of one operation on
 * fp32 operands: equals the correctly rounded fp32 operation. */
static inline double rnd(int f32, double x) { return f32 ? (double)(float)x : x; }

/*
 * dW, dD: fp64 outputs, flat over projections like W.  dW = -tau_s SU,
 * dD = -dt SD (per step of delay), summed over the batch (g carries 1/B).
 * stats[0] = degenerate crossings (I- <= theta) whose jump was skipped.
 */
int oracle_backward(int L, const int* n, const int* kind, const int* rec,
                    float tau_m, float tau_s, float theta, float dt, int max_delay, const int* pmax,
                    int B, int T, int loss, float readout_scale,
                    const int* in_off, const int* in_step, const int* in_neuron,
                    const float* W, const float* D, int cap,
                    const int* rec_count, const int* rec_step, const int* rec_neuron,
                    const float* rec_I, const float* g, const int* nstar,
                    const double* rec_dlp, int mode,
                    double* dW, double* dD, long* stats) {
    topo_t t;
    int rc = build_topo(&t, L, n, kind, rec);
    if (rc) return rc;
    if (max_delay < 0 || max_delay > 255 || cap < 0 || (mode != 0 && mode != 1)) return OR_EINVAL;
    if (loss != OR_LOSS_CE_SUM && loss != OR_LOSS_CE_MAX && loss != OR_LOSS_DMSE) return OR_EINVAL;
    if ((loss == OR_LOSS_DMSE) != (t.kind[L - 1] == OR_LIF)) return OR_EINVAL;
    rc = check_inputs(&t, B, T, in_off, in_step, in_neuron);
    if (rc) return rc;
    for (int li = 0; li < t.n_lif; ++li)
        for (int b = 0; b < B; ++b)
            if (rec_count[(size_t)li * B + b] > cap) return OR_EOVERFLOW;
    const int f32 = (mode == 1);
    double alpha, beta, cc;
    if (f32) {
        float k4[4];
        rc = oracle_constants(tau_m, tau_s, dt, k4);
        if (rc) return rc;
        alpha = k4[0]; beta = k4[1]; cc = k4[3];
    } else {
        if (!(dt > 0.0f) || tau_m == tau_s) return OR_EINVAL;
        alpha = exp(-(double)dt / (double)tau_m);
        beta = exp(-(double)dt / (double)tau_s);
        cc = (double)tau_m / ((double)tau_m - (double)tau_s) * (alpha - beta);
    }
    const int C = t.n[L - 1];
    const int out_l = L - 1;

    long clamped = 0, degenerate = 0;
    unsigned char* slot = (unsigned char*)malloc((size_t)t.n_params);
    double* SU = (double*)calloc((size_t)t.n_params, sizeof(double));
    double* SD = (double*)calloc((size_t)t.n_params, sizeof(double));
    double* lv = (double*)malloc(sizeof(double) * t.n_state);
    double* lI = (double*)malloc(sizeof(double) * t.n_state);
    double* H = (double*)malloc(sizeof(double) * 2 * (size_t)T * t.n_state);
    double* A = (double*)malloc(sizeof(double) * t.n_state);
    double* src = (double*)malloc(sizeof(double) * C);
    if (!slot || !SU || !SD || !lv || !lI || !H || !A || !src) {
        free(slot); free(SU); free(SD); free(lv); free(lI); free(H); free(A); free(src);
        return OR_ENOMEM;
    }
    if (fill_slots(&t, D, max_delay, pmax, slot, &clamped)) {
        free(slot); free(SU); free(SD); free(lv); free(lI); free(H); free(A); free(src);
        return OR_EINVAL;
    }

    int rec_hi[OR_MAXL];
    for (int b = 0; b < B; ++b) {
        memset(lv, 0, sizeof(double) * t.n_state);
        memset(lI, 0, sizeof(double) * t.n_state);
        for (int k = 0; k < C && loss != OR_LOSS_DMSE; ++k) {
            const double gk = (double)g[(size_t)b * C + k];
            const double sk = (loss == OR_LOSS_CE_SUM) ? (double)readout_scale * gk / (double)tau_m
                                                       : gk / (double)tau_m;
            src[k] = f32 ? (double)(float)sk : sk;
        }
        for (int l = 0; l < L; ++l)
            if (t.lif_idx[l] >= 0) rec_hi[l] = rec_count[(size_t)t.lif_idx[l] * B + b];
        for (int n_ = T - 1; n_ >= 0; --n_) {
            /* 1. adjoint free dynamics over one step */
            if (n_ <= T - 2) {
                for (int s = 0; s < t.n_state; ++s) {
                    const double v = lv[s];
                    lI[s] = rnd(f32, rnd(f32, beta * lI[s]) + rnd(f32, cc * v));
                    lv[s] = rnd(f32, alpha * v);
                }
            }
            /* 2. the "+" values at this step */
            double* h = H + 2 * (size_t)n_ * t.n_state;
            for (int s = 0; s < t.n_state; ++s) {
                h[2 * s] = lv[s];
                h[2 * s + 1] = lI[s];
            }
            /* 3. loss source on the LI readout */
            for (int k = 0; k < C && loss != OR_LOSS_DMSE; ++k) {
                const int s = t.st_off[out_l] + k;
                if (loss == OR_LOSS_CE_SUM || nstar[(size_t)b * C + k] == n_)
                    lv[s] = rnd(f32, lv[s] - src[k]);
            }
            /* 4. LIF spikes at this step: delayed postsynaptic sums, jumps */
            int rec_lo[OR_MAXL];
            for (int l = 1; l < L; ++l) {
                if (t.lif_idx[l] < 0) continue;
                const size_t base = (size_t)t.lif_idx[l] * B * cap + (size_t)b * cap;
                int lo = rec_hi[l];
                while (lo > 0 && rec_step[base + lo - 1] == n_) --lo;
                rec_lo[l] = lo;
                for (int k = lo; k < rec_hi[l]; ++k) A[t.st_off[l] + rec_neuron[base + k]] = 0.0;
            }
            for (int p = 0; p < t.P; ++p) {
                const int a = t.pre[p], q = t.post[p];
                if (a == 0) continue;
                const int nq = t.n[q];
                const size_t base = (size_t)t.lif_idx[a] * B * cap + (size_t)b * cap;
                for (int k = rec_lo[a]; k < rec_hi[a]; ++k) {
                    const int i = rec_neuron[base + k];
                    const long row = t.w_off[p] + (long)i * nq;
                    double Ai = 0.0;
                    for (int j = 0; j < nq; ++j) {
                        const int m = n_ + slot[row + j];
                        if (m > T - 1) continue;
                        const double* hv = H + 2 * ((size_t)m * t.n_state + t.st_off[q] + j);
                        const double d = rnd(f32, hv[1] - hv[0]);
                        Ai = rnd(f32, Ai - rnd(f32, (double)W[row + j] * d));
                    }
                    A[t.st_off[a] + i] = rnd(f32, A[t.st_off[a] + i] + Ai);
                }
            }
            for (int l = 1; l < L; ++l) {
                if (t.lif_idx[l] < 0) continue;
                const size_t base = (size_t)t.lif_idx[l] * B * cap + (size_t)b * cap;
                for (int k = rec_lo[l]; k < rec_hi[l]; ++k) {
                    const int s = t.st_off[l] + rec_neuron[base + k];
                    const double den = rnd(f32, (double)rec_I[base + k] - (double)theta);
                    if (den > 0.0) {
                        double num = rnd(f32, rnd(f32, (double)theta * lv[s]) + A[s]);
                        if (rec_dlp) num = rnd(f32, num + rec_dlp[base + k]);
                        lv[s] = rnd(f32, lv[s] + rnd(f32, num / den));
                    } else {
                        ++degenerate;
                    }
                }
                rec_hi[l] = rec_lo[l];
            }
        }
        /* gradient sums over this sample's spikes, in spike order */
        for (int p = 0; p < t.P; ++p) {
            const int a = t.pre[p], q = t.post[p];
            const int nq = t.n[q];
            const int cnt = (a == 0) ? in_off[b + 1] - in_off[b] : rec_count[(size_t)t.lif_idx[a] * B + b];
            const size_t base = (a == 0) ? (size_t)in_off[b] : (size_t)t.lif_idx[a] * B * cap + (size_t)b * cap;
            for (int k = 0; k < cnt; ++k) {
                const int i = (a == 0) ? in_neuron[base + k] : rec_neuron[base + k];
                const int n0 = (a == 0) ? in_step[base + k] : rec_step[base + k];
                const long row = t.w_off[p] + (long)i * nq;
                for (int j = 0; j < nq; ++j) {
                    const int m = n0 + slot[row + j];
                    if (m > T - 1) continue;
                    const double* hv = H + 2 * ((size_t)m * t.n_state + t.st_off[q] + j);
                    const double v = hv[0], u = hv[1];
                    const double d = rnd(f32, u - v);
                    const double wd = rnd(f32, (double)W[row + j] * d);
                    SU[row + j] = rnd(f32, SU[row + j] + u);
                    SD[row + j] = rnd(f32, SD[row + j] + wd);
                }
            }
        }
    }
    for (long k = 0; k < t.n_params; ++k) {
        dW[k] = -(double)tau_s * SU[k];
        dD[k] = -(double)dt * SD[k];
    }
    if (stats) stats[0] = degenerate;
    free(slot); free(SU); free(SD); free(lv); free(lI); free(H); free(A); free(src);
    return OR_OK;
}
