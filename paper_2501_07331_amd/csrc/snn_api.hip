// Host side of libsnn: validation, scratch sizing, LDS planning, launch
// sequencing and the status read-back.  See include/snn.h for the contract.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>

#include "snn_internal.h"

namespace {

constexpr size_t kLdsPerGroup = 160 * 1024;   // gfx950: 160 KiB of LDS per workgroup

}  // namespace

struct snn_net {
    Topo t;
    float tau_m, tau_s, theta, dt;
    int max_delay;
    int threads;
    size_t lds;                 // dynamic LDS bytes of the persistent kernels
    int extra_off;              // byte offset of the masks / fp64 jump sums
    hipStream_t stream;
    long long n_params;
    long long cnt[SNN_MAXP];
    int n_state;
    int st_off[SNN_MAX_LAYERS];
    // device scratch
    uint8_t* slot;
    float* ring[SNN_MAX_LAYERS];
    int* in_idx;
    int* rec_n;
    float* rec_I;
    float* rec_D;
    int* rec_idx;
    float* z;
    int* nstar;
    float* src;
    float* Vf;
    float* If;
    double* SU;
    double* SD;
    DevStatus* st;
    DevStatus* st_host;         // pinned
    // the last forward's inputs, kept for the backward
    const float* W[SNN_MAXP];
    const int* in_neuron;
    int fwd_ok, fwd_overflow;
    int timing;
    hipEvent_t ev[6];           // around the forward, backward A, backward B kernels
    snn_stats stats;
    char err[256];
};

static int fail(snn_net* net, int code, const char* fmt, ...) {
    if (net) {
        va_list ap;
        va_start(ap, fmt);
        vsnprintf(net->err, sizeof(net->err), fmt, ap);
        va_end(ap);
    }
    return code;
}

#define HIP_TRY(net, expr)                                                                       \
    do {                                                                                         \
        hipError_t e_ = (expr);                                                                  \
        if (e_ != hipSuccess)                                                                    \
            return fail((net), SNN_EDEVICE, "%s: %s", #expr, hipGetErrorString(e_));            \
    } while (0)

static void free_all(snn_net* n) {
    void* bufs[] = {n->slot, n->in_idx, n->rec_n, n->rec_I, n->rec_D, n->rec_idx, n->z, n->nstar,
                    n->src, n->Vf, n->If, n->SU, n->SD, n->st};
    for (void* p : bufs)
        if (p) (void)hipFree(p);
    for (int l = 0; l < SNN_MAX_LAYERS; ++l)
        if (n->ring[l]) (void)hipFree(n->ring[l]);
    if (n->st_host) (void)hipHostFree(n->st_host);
    for (int i = 0; i < 6; ++i)
        if (n->ev[i]) (void)hipEventDestroy(n->ev[i]);
}

template <typename T>
static hipError_t dalloc(T** p, size_t count) {
    *p = nullptr;
    if (count == 0) count = 1;
    return hipMalloc((void**)p, count * sizeof(T));
}

extern "C" int snn_create(const snn_layer* layers, int32_t n_layers, float tau_m, float tau_s,
                          float theta, float dt, int32_t max_delay, const snn_opts* opts,
                          snn_net** out) {
    if (!out) return SNN_EINVAL;
    *out = nullptr;
    if (!layers || !opts) return SNN_EINVAL;
    if (n_layers < 2 || n_layers > SNN_MAX_LAYERS) return SNN_EINVAL;
    if (!(dt > 0.0f) || !(tau_m > 0.0f) || !(tau_s > 0.0f) || tau_m == tau_s) return SNN_EINVAL;
    if (!(theta == theta)) return SNN_EINVAL;
    if (max_delay < 0 || max_delay > SNN_MAX_DELAY) return SNN_EINVAL;
    if (opts->batch < 1 || opts->T < 1 || opts->record_capacity < 0) return SNN_EINVAL;
    if (opts->loss != SNN_LOSS_CE_SUM && opts->loss != SNN_LOSS_CE_MAX) return SNN_EINVAL;
    if (opts->flags & ~(SNN_FLAG_HBM_RINGS | SNN_FLAG_TIMING)) return SNN_EINVAL;
    for (int l = 0; l < n_layers; ++l) {
        const snn_layer& y = layers[l];
        if (y.n < 1) return SNN_EINVAL;
        if (l == 0 && y.kind != SNN_INPUT) return SNN_EINVAL;
        if (l > 0 && l < n_layers - 1 && y.kind != SNN_LIF) return SNN_EINVAL;
        if (l == n_layers - 1 && y.kind != SNN_LI) return SNN_EINVAL;
        if (y.recurrent && y.kind != SNN_LIF) return SNN_EINVAL;
        if (l > 0 && y.n > SNN_MAX_NEURONS) return SNN_EINVAL;
    }
    if ((long long)opts->batch * (opts->T + 1) > (1LL << 31)) return SNN_EINVAL;

    snn_net* net = (snn_net*)calloc(1, sizeof(snn_net));
    if (!net) return SNN_ENOMEM;
    Topo& t = net->t;
    t.L = n_layers;
    t.B = opts->batch;
    t.T = opts->T;
    t.S = max_delay + 1;
    t.cap = opts->record_capacity;
    t.loss = opts->loss;
    t.n_in = layers[0].n;
    t.rscale = opts->readout_scale;
    t.theta = theta;
    t.tau_s = tau_s;
    t.dt = dt;
    // exact one-step propagators of Table 1's free dynamics, fp64 on the host
    const double a = exp(-(double)dt / (double)tau_m);
    const double bb = exp(-(double)dt / (double)tau_s);
    t.alpha = (float)a;
    t.beta = (float)bb;
    t.gamma = (float)((double)tau_s / ((double)tau_s - (double)tau_m) * (bb - a));
    t.cc = (float)((double)tau_m / ((double)tau_m - (double)tau_s) * (a - bb));
    net->tau_m = tau_m;
    net->tau_s = tau_s;
    net->theta = theta;
    net->dt = dt;
    net->max_delay = max_delay;
    net->stream = (hipStream_t)opts->hip_stream;

    int maxn = 0, so = 0;
    for (int l = 0; l < n_layers; ++l) {
        t.n[l] = layers[l].n;
        t.kind[l] = layers[l].kind;
        t.lif[l] = -1;
        t.lif_off[l] = 0;
        t.ring_lds[l] = -1;
        net->st_off[l] = so;
        if (l > 0) {
            so += layers[l].n;
            maxn = std::max(maxn, layers[l].n);
        }
        if (layers[l].kind == SNN_LIF) {
            t.lif[l] = t.n_lif++;
            t.lif_off[l] = t.lif_total;
            t.lif_total += layers[l].n;
        }
    }
    net->n_state = so;
    long long off = 0;
    for (int l = 1; l < n_layers; ++l) {
        for (int r = 0; r < 1 + (layers[l].recurrent ? 1 : 0); ++r) {
            const int p = t.P++;
            t.pre[p] = r ? l : l - 1;
            t.post[p] = l;
            t.woff[p] = off;
            net->cnt[p] = (long long)t.n[t.pre[p]] * t.n[l];
            off += net->cnt[p];
        }
    }
    net->n_params = off;
    net->threads = ((maxn + 63) / 64) * 64;
    const int nwaves = net->threads / 64;

    // LDS plan: ballot masks (forward) or fp64 jump sums (backward A) after the
    // rings; LIF rings first (they carry most events), then the readout ring.
    const size_t masks = (size_t)2 * t.n_lif * nwaves * sizeof(unsigned long long);
    const size_t accs = (size_t)2 * t.lif_total * sizeof(double);
    const size_t extra = (std::max(masks, accs) + 15) & ~(size_t)15;
    size_t ring_bytes = 0;
    for (int pass = 0; pass < 2; ++pass) {
        for (int l = 1; l < n_layers; ++l) {
            const bool want = (pass == 0) ? (t.kind[l] == SNN_LIF) : (t.kind[l] == SNN_LI);
            if (!want) continue;
            const size_t bytes = (size_t)t.S * t.n[l] * sizeof(float);
            if (!(opts->flags & SNN_FLAG_HBM_RINGS) && ring_bytes + bytes + extra <= kLdsPerGroup) {
                t.ring_lds[l] = (int)(ring_bytes / sizeof(float));
                ring_bytes += bytes;
            }
        }
    }
    ring_bytes = (ring_bytes + 15) & ~(size_t)15;
    net->extra_off = (int)ring_bytes;
    net->lds = ring_bytes + extra;

    hipError_t e = hipSuccess;
    const size_t B = t.B, T1 = (size_t)t.T + 1, cap = (size_t)t.cap, nl = (size_t)std::max(t.n_lif, 1);
    const size_t C = t.n[n_layers - 1];
#define ALLOC(ptr, count)                                 \
    if (e == hipSuccess) e = dalloc(&(ptr), (count));
    ALLOC(net->slot, (size_t)net->n_params);
    for (int l = 1; l < n_layers; ++l)
        if (t.ring_lds[l] < 0) ALLOC(net->ring[l], B * t.S * t.n[l]);
    ALLOC(net->in_idx, B * T1);
    ALLOC(net->rec_n, nl * B * cap);
    ALLOC(net->rec_I, nl * B * cap);
    ALLOC(net->rec_D, nl * B * cap);
    ALLOC(net->rec_idx, nl * B * T1);
    ALLOC(net->z, B * C);
    ALLOC(net->nstar, B * C);
    ALLOC(net->src, B * C);
    ALLOC(net->Vf, B * so);
    ALLOC(net->If, B * so);
    ALLOC(net->SU, (size_t)net->n_params);
    ALLOC(net->SD, (size_t)net->n_params);
    ALLOC(net->st, 1);
#undef ALLOC
    if (e == hipSuccess) e = hipHostMalloc((void**)&net->st_host, sizeof(DevStatus), hipHostMallocDefault);
    if (e == hipSuccess) e = set_kernel_lds_limits(std::max(net->lds, (size_t)1));
    net->timing = (opts->flags & SNN_FLAG_TIMING) ? 1 : 0;
    for (int i = 0; i < 6 && net->timing && e == hipSuccess; ++i) e = hipEventCreate(&net->ev[i]);
    if (e != hipSuccess) {
        const int code = (e == hipErrorOutOfMemory) ? SNN_ENOMEM : SNN_EDEVICE;
        free_all(net);
        free(net);
        return code;
    }
    *out = net;
    return SNN_OK;
}

extern "C" int snn_num_projections(const snn_net* net, int32_t* n) {
    if (!net || !n) return SNN_EINVAL;
    *n = net->t.P;
    return SNN_OK;
}

extern "C" int snn_projection_info(const snn_net* net, int32_t p, int32_t* pre_layer,
                                   int32_t* post_layer, int32_t* n_pre, int32_t* n_post) {
    if (!net || p < 0 || p >= net->t.P) return SNN_EINVAL;
    if (pre_layer) *pre_layer = net->t.pre[p];
    if (post_layer) *post_layer = net->t.post[p];
    if (n_pre) *n_pre = net->t.n[net->t.pre[p]];
    if (n_post) *n_post = net->t.n[net->t.post[p]];
    return SNN_OK;
}

static int read_status(snn_net* net) {
    HIP_TRY(net, hipMemcpyAsync(net->st_host, net->st, sizeof(DevStatus), hipMemcpyDeviceToHost,
                                net->stream));
    HIP_TRY(net, hipStreamSynchronize(net->stream));
    return SNN_OK;
}

extern "C" int snn_forward(snn_net* net, const snn_spikes_in* in, const float* const* W,
                           const float* const* D, const int32_t* labels, snn_spikes_out* records,
                           float* loss, float* z) {
    if (!net) return SNN_EINVAL;
    net->err[0] = 0;
    net->fwd_ok = 0;
    Topo& t = net->t;
    if (!in || !in->offsets || (in->nnz > 0 && (!in->step || !in->neuron)) || in->nnz < 0)
        return fail(net, SNN_EINVAL, "input spikes: NULL pointer or negative nnz");
    if (!W || !D || !labels || !loss) return fail(net, SNN_EINVAL, "NULL W, D, labels or loss");
    for (int p = 0; p < t.P; ++p)
        if (!W[p] || !D[p]) return fail(net, SNN_EINVAL, "NULL W or D of projection %d", p);
    if (t.n_lif > 0 && !records) return fail(net, SNN_EINVAL, "NULL records");
    for (int l = 1; l < t.L; ++l) {
        if (t.kind[l] != SNN_LIF) continue;
        const snn_spikes_out& r = records[t.lif[l]];
        if (!r.count || (t.cap > 0 && (!r.step || !r.neuron)))
            return fail(net, SNN_EINVAL, "NULL record buffers of layer %d", l);
    }
    hipStream_t s = net->stream;
    const int C = t.n[t.L - 1];
    HIP_TRY(net, launch_reset_status(net->st, s));
    HIP_TRY(net, launch_validate(in->offsets, in->step, in->neuron, in->nnz, t.B, t.T, t.n_in, labels,
                                 C, net->st, s));
    HIP_TRY(net, launch_step_index(in->offsets, in->step, t.B, t.T, net->in_idx, net->st, s));
    HIP_TRY(net, launch_round_delays(D, t.woff, net->cnt, t.P, net->max_delay, net->slot, net->st, s));

    FwdArgs a{};
    a.t = t;
    for (int p = 0; p < t.P; ++p) a.W[p] = W[p];
    a.slot = net->slot;
    for (int l = 0; l < SNN_MAX_LAYERS; ++l) a.ring[l] = net->ring[l];
    a.in_neuron = in->neuron;
    a.in_idx = net->in_idx;
    for (int l = 1; l < t.L; ++l) {
        if (t.kind[l] != SNN_LIF) continue;
        a.out_count[l] = records[t.lif[l]].count;
        a.out_step[l] = records[t.lif[l]].step;
        a.out_neuron[l] = records[t.lif[l]].neuron;
    }
    a.rec_n = net->rec_n;
    a.rec_I = net->rec_I;
    a.rec_idx = net->rec_idx;
    a.z = net->z;
    a.nstar = net->nstar;
    a.Vf = net->Vf;
    a.If = net->If;
    a.st = net->st;
    a.mask_off = net->extra_off;
    if (net->timing) HIP_TRY(net, hipEventRecord(net->ev[0], s));
    HIP_TRY(net, launch_forward(a, net->threads, net->lds, s));
    if (net->timing) HIP_TRY(net, hipEventRecord(net->ev[1], s));
    HIP_TRY(net, launch_loss(net->z, labels, net->nstar, t.B, C, t.loss, t.rscale, net->tau_m, loss,
                             net->src, net->st, s));
    if (z)
        HIP_TRY(net, hipMemcpyAsync(z, net->z, sizeof(float) * t.B * C, hipMemcpyDeviceToDevice, s));
    int rc = read_status(net);
    if (rc) return rc;
    const DevStatus& h = *net->st_host;
    if (h.bad_input)
        return fail(net, SNN_EINVAL, "input spikes or labels invalid (offsets, range, order)");
    memset(&net->stats, 0, sizeof(net->stats));
    net->stats.input_spikes = in->nnz;
    net->stats.clamped_delays = (int64_t)h.clamped;
    net->stats.overflow = h.overflow;
    for (int l = 1; l < t.L; ++l)
        if (t.ring_lds[l] >= 0) net->stats.lds_rings |= 1 << l;
    long long ev = 0;
    for (int p = 0; p < t.P; ++p) {
        const int pre = t.pre[p];
        const long long spikes = (pre == 0) ? in->nnz : (long long)h.layer_spikes[t.lif[pre]];
        ev += spikes * t.n[t.post[p]];
    }
    for (int li = 0; li < t.n_lif; ++li) net->stats.lif_spikes += (int64_t)h.layer_spikes[li];
    net->stats.events = ev;
    if (net->timing) HIP_TRY(net, hipEventElapsedTime(&net->stats.forward_kernel_ms, net->ev[0], net->ev[1]));
    for (int p = 0; p < t.P; ++p) net->W[p] = W[p];
    net->in_neuron = in->neuron;
    net->fwd_ok = 1;
    net->fwd_overflow = h.overflow;
    if (h.overflow) return fail(net, SNN_EOVERFLOW, "a sample exceeded record_capacity spikes");
    return SNN_OK;
}

extern "C" int snn_backward(snn_net* net, float* const* dW, float* const* dD) {
    if (!net) return SNN_EINVAL;
    net->err[0] = 0;
    Topo& t = net->t;
    if (!net->fwd_ok) return fail(net, SNN_ESTATE, "snn_backward without a successful snn_forward");
    if (net->fwd_overflow)
        return fail(net, SNN_EOVERFLOW, "the last forward overflowed its spike records");
    if (!dW || !dD) return fail(net, SNN_EINVAL, "NULL dW or dD");
    for (int p = 0; p < t.P; ++p)
        if (!dW[p] || !dD[p]) return fail(net, SNN_EINVAL, "NULL dW or dD of projection %d", p);
    hipStream_t s = net->stream;
    HIP_TRY(net, launch_fill_f64(net->SU, net->n_params, s));
    HIP_TRY(net, launch_fill_f64(net->SD, net->n_params, s));
    BwdArgs a{};
    a.t = t;
    for (int p = 0; p < t.P; ++p) a.W[p] = net->W[p];
    a.slot = net->slot;
    for (int l = 0; l < SNN_MAX_LAYERS; ++l) a.ring[l] = net->ring[l];
    a.in_neuron = net->in_neuron;
    a.in_idx = net->in_idx;
    a.rec_n = net->rec_n;
    a.rec_I = net->rec_I;
    a.rec_D = net->rec_D;
    a.rec_idx = net->rec_idx;
    a.src = net->src;
    a.nstar = net->nstar;
    a.SU = net->SU;
    a.SD = net->SD;
    a.st = net->st;
    a.acc_off = net->extra_off;
    if (net->timing) HIP_TRY(net, hipEventRecord(net->ev[2], s));
    HIP_TRY(net, launch_backward_a(a, net->threads, net->lds, s));
    if (net->timing) HIP_TRY(net, hipEventRecord(net->ev[3], s));
    HIP_TRY(net, launch_backward_b(a, net->threads, net->lds, s));
    if (net->timing) HIP_TRY(net, hipEventRecord(net->ev[4], s));
    HIP_TRY(net, launch_finalize(net->SU, net->SD, dW, dD, t.woff, net->cnt, t.P, t.tau_s, t.dt, s));
    int rc = read_status(net);
    if (rc) return rc;
    net->stats.degenerate_jumps = (int64_t)net->st_host->degenerate;
    if (net->timing) {
        HIP_TRY(net, hipEventElapsedTime(&net->stats.backward_a_ms, net->ev[2], net->ev[3]));
        HIP_TRY(net, hipEventElapsedTime(&net->stats.backward_b_ms, net->ev[3], net->ev[4]));
    }
    return SNN_OK;
}

extern "C" int snn_get_state(const snn_net* net, int32_t layer, float* V, float* I) {
    if (!net || layer < 1 || layer >= net->t.L || !V || !I) return SNN_EINVAL;
    if (!net->fwd_ok) return SNN_ESTATE;
    snn_net* m = const_cast<snn_net*>(net);
    const Topo& t = net->t;
    HIP_TRY(m, launch_copy_state(net->Vf, net->n_state, net->st_off[layer], t.n[layer], t.B, V,
                                 net->stream));
    HIP_TRY(m, launch_copy_state(net->If, net->n_state, net->st_off[layer], t.n[layer], t.B, I,
                                 net->stream));
    HIP_TRY(m, hipStreamSynchronize(net->stream));
    return SNN_OK;
}

extern "C" int snn_get_stats(const snn_net* net, snn_stats* out) {
    if (!net || !out) return SNN_EINVAL;
    *out = net->stats;
    return SNN_OK;
}

extern "C" const char* snn_last_error(const snn_net* net) { return net ? net->err : "NULL handle"; }

extern "C" void snn_destroy(snn_net* net) {
    if (!net) return;
    (void)hipStreamSynchronize(net->stream);
    free_all(net);
    free(net);
}
