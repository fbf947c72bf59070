// Host side of libsnn: validation, scratch sizing, LDS planning, launch
// sequencing and the status read-back.  See include/snn.h for the contract.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <mutex>

#include "snn_internal.h"

// Fixed device scratch of snn_backward_noalloc: one copy per device, held
// until the process ends.  Host code never uses this name as an address (on
// the host it is only a stand-in for the symbol): the device address comes
// from hipGetSymbolAddress, once per device, in snn_create.
constexpr long long kScratchInts = (long long)(SNN_NOALLOC_SCRATCH_BYTES / sizeof(int));
static __device__ __align__(256) int scratch[kScratchInts];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
int* g_scratch_addr[kMaxDevices];   // device address of `scratch` per device, NULL until looked up

// The address of `scratch` on the current device (looked up on first use).
hipError_t scratch_address(int** out) {
    *out = nullptr;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_addr[dev]) {
        void* ptr = nullptr;
        e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        g_scratch_addr[dev] = static_cast<int*>(ptr);
    }
    *out = g_scratch_addr[dev];
    return hipSuccess;
}
}  // namespace

namespace {

constexpr size_t kLds = 160 * 1024;   // gfx950: 160 KiB of LDS per workgroup
constexpr int kGroupStage = 16384;    // spikes of a sample the grouping stages in LDS (32 KiB)
enum { K_SCAN, K_CORE, K_READ, K_RADJ, K_BCORE, K_GROUP, K_GRAD, K_N };

size_t align16(size_t x) { return (x + 15) & ~(size_t)15; }

}  // namespace

struct snn_net {
    Topo t;
    float tau_m, tau_s, theta, dt;
    double alpha64, beta64, cc64;   // backward propagators, fp64
    int reg_on;                     // spike-count regulariser on some LIF layer
    double reg_rho[SNN_MAX_LIF];    // its strength per LIF layer
    double reg_nu;                  // its target spikes per neuron and sample
    int* ncount;                    // [lif_total] spikes per neuron over the batch
    double* nterm;                  // [lif_total] regulariser jump term per neuron
    float dmse_delta;
    int max_delay;
    int core_threads;           // LIF-core workgroup size (without a fused readout wave)
    int ro_fused, ro_off;       // the LI readout runs as one more wave of the forward core
    int read_threads;           // readout workgroup size
    size_t lds_core_f, lds_core_b, lds_scan, lds_read, lds_grad, lds_radj;
    int mask_off, ids_off, scan_tb, table_lds;
    int bpart_off;              // backward-core LDS plan
    int bring_mode[SNN_MAX_LAYERS];   // adjoint ring of a LIF layer: -2 none, -1 HBM, >= 0 LDS
                                      // byte offset
    int radj_threads, radj_tab;
    // cluster mode of the LIF cores (see ClusterArgs): on for the forward /
    // backward core, workgroups per sample, samples per launch, most
    // LIF-post projections of a LIF layer, the backward's staging offset,
    // the next exchange tag (odd) and the exchange words
    int cl_f, cl_b, cl_G, cl_spp_f, cl_spp_b, cl_np, cl_off_b;
    int cl_threads;             // workgroup: the neuron wave and one wave per LIF -> LIF projection
    unsigned cl_tag;
    unsigned long long* clx;
    int grad_J, grad_TW, grad_KL, grad_threads, grad_SB, grad_bs, grad_nblk, grad_ngroups, grad_spcap,
        grad_glcap;
    GradGroup grad_grp[SNN_MAX_LAYERS];
    hipStream_t stream;
    hipStream_t aux;                   // second stream: spike grouping beside the backward sweep
    hipEvent_t fork, join;             // its start after the caller's work, its end before gradients
    long long n_params;
    long long cnt[SNN_MAXP];
    int n_state;
    int st_off[SNN_MAX_LAYERS];
    // device scratch
    uint8_t* slot;
    uint2* ws;                  // (weight bits, slot) of every synapse
    int* steptab;
    int* in_idx;
    float* A_in;
    float* fring[SNN_MAXP];
    double* bring[SNN_MAX_LAYERS];
    int* rec_n;
    int* rec_s;
    float* rec_I;
    int* rec_idx;
    int* rec_cnt;
    int* rec_goff;
    unsigned short* rec_gstep;
    float* z;
    int* nstar;
    double* src;
    float* Vf;
    float* If;
    float* table;
    double2* tr_lif;            // adjoint trajectories (lambda_I, lambda_I - lambda_V) [B][T][N]
    double2* tr_out;
    double* A2;
    double* gpart;
    float* mom;                 // Adam moments [4][n_params], allocated by the first Adam step
    double* xlp_out;            // spike-time loss: jump terms of the output layer's records [B][cap]
    double* jx[SNN_MAX_LIF];    // per LIF layer: jump terms with the caller's dl_p/dt [B][cap]
    int ran[K_N];               // kernels enqueued (and timed) by the last call
    long long adam_steps;
    int* in_goff;
    unsigned short* in_gstep;
    long long in_gstep_cap;
    int* scratch;               // device address of the fixed scratch (snn_backward_noalloc)
    DevStatus* st;
    DevStatus* st_host;         // pinned
    // the last forward's inputs, kept for the backward
    const float* W[SNN_MAXP];
    const int* in_off;
    const int* in_step;
    const int* in_neuron;
    int in_nnz;
    int fwd_ok, fwd_overflow;
    int timing;
    hipEvent_t ev[2 * K_N];
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

// Entries per LIF layer of the grouped spike steps (16-bit).
static size_t gstep_stride(size_t B, size_t cap) { return (B * cap + 7) & ~(size_t)7; }

static void free_all(snn_net* n) {
    void* bufs[] = {n->slot,    n->in_idx,  n->A_in,     n->rec_n,     n->rec_s,  n->rec_I,
                    n->rec_idx, n->rec_cnt, n->rec_goff, n->rec_gstep, n->z,      n->nstar,
                    n->src,     n->Vf,      n->If,       n->table,     n->tr_lif, n->tr_out,
                    n->A2,       n->in_goff,   n->in_gstep, n->st,
                    n->gpart,   n->ws,      n->steptab, n->mom,   n->xlp_out, n->ncount,
                    n->nterm,   n->clx};
    for (void* p : bufs)
        if (p) (void)hipFree(p);
    for (int p = 0; p < SNN_MAXP; ++p)
        if (n->fring[p]) (void)hipFree(n->fring[p]);
    for (int l = 0; l < SNN_MAX_LAYERS; ++l)
        if (n->bring[l]) (void)hipFree(n->bring[l]);
    for (int l = 0; l < SNN_MAX_LIF; ++l)
        if (n->jx[l]) (void)hipFree(n->jx[l]);
    if (n->st_host) (void)hipHostFree(n->st_host);
    for (int i = 0; i < 2 * K_N; ++i)
        if (n->ev[i]) (void)hipEventDestroy(n->ev[i]);
    if (n->fork) (void)hipEventDestroy(n->fork);
    if (n->join) (void)hipEventDestroy(n->join);
    if (n->aux) (void)hipStreamDestroy(n->aux);
}

template <typename T>
static hipError_t dalloc(T** p, size_t count) {
    *p = nullptr;
    if (count == 0) count = 1;
    return hipMalloc((void**)p, count * sizeof(T));
}

// reason of the last failed snn_create on this thread
static thread_local char g_create_err[256] = "";

extern "C" int snn_create(const snn_layer* layers, int32_t n_layers, float tau_m, float tau_s,
                          float theta, float dt, int32_t max_delay, const snn_opts* opts,
                          snn_net** out) {
    g_create_err[0] = '\0';
    if (!out) return SNN_EINVAL;
    *out = nullptr;
    if (!layers || !opts) return SNN_EINVAL;
    if (n_layers < 2 || n_layers > SNN_MAX_LAYERS) return SNN_EINVAL;
    if (!(dt > 0.0f) || !(tau_m > 0.0f) || !(tau_s > 0.0f) || tau_m == tau_s) return SNN_EINVAL;
    if (!(theta == theta)) return SNN_EINVAL;
    if (max_delay < 0 || max_delay > SNN_MAX_DELAY) return SNN_EINVAL;
    if (opts->batch < 1 || opts->T < 1 || opts->record_capacity < 0) return SNN_EINVAL;
    if (opts->loss != SNN_LOSS_CE_SUM && opts->loss != SNN_LOSS_CE_MAX &&
        opts->loss != SNN_LOSS_DMSE)
        return SNN_EINVAL;
    const bool dmse = opts->loss == SNN_LOSS_DMSE;
    if (dmse && (!(opts->dmse_delta == opts->dmse_delta) || isinf(opts->dmse_delta) ||
                 opts->record_capacity < 1))
        return SNN_EINVAL;
    if (opts->flags &
        ~(SNN_FLAG_HBM_RINGS | SNN_FLAG_TIMING | SNN_FLAG_SEPARATE_READOUT | SNN_FLAG_CLUSTER))
        return SNN_EINVAL;
    if (opts->reg_strength && (!(opts->reg_target >= 0.0f) || isinf(opts->reg_target)))
        return SNN_EINVAL;
    for (int l = 0; l < n_layers; ++l) {
        const snn_layer& y = layers[l];
        if (y.n < 1) return SNN_EINVAL;
        if (l == 0 && (y.kind != SNN_INPUT || y.n > SNN_MAX_INPUT)) return SNN_EINVAL;
        if (l > 0 && l < n_layers - 1 && y.kind != SNN_LIF) return SNN_EINVAL;
        if (l == n_layers - 1 && y.kind != (dmse ? SNN_LIF : SNN_LI)) return SNN_EINVAL;
        if (y.recurrent && (y.kind != SNN_LIF || l == n_layers - 1)) return SNN_EINVAL;
        if (l > 0 && y.n > SNN_MAX_NEURONS) return SNN_EINVAL;
    }
    // the kernels hold per-LIF-layer state for at most SNN_MAX_LIF layers
    if (dmse && n_layers - 1 > SNN_MAX_LIF) return SNN_EINVAL;
    // spike steps are staged as 16-bit values in the gradient pass
    if (opts->T > SNN_MAX_T) return SNN_EINVAL;
    if ((long long)opts->batch * (opts->T + 1) > (1LL << 31)) return SNN_EINVAL;

    snn_net* net = (snn_net*)calloc(1, sizeof(snn_net));
    if (!net) return SNN_ENOMEM;
    Topo& t = net->t;
    t.L = n_layers;
    t.B = opts->batch;
    t.T = opts->T;
    t.S = max_delay + 1;     // per projection below
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
    net->alpha64 = a;
    net->beta64 = bb;
    net->cc64 = (double)tau_m / ((double)tau_m - (double)tau_s) * (a - bb);
    net->tau_m = tau_m;
    net->tau_s = tau_s;
    net->theta = theta;
    net->dt = dt;
    net->max_delay = max_delay;
    net->dmse_delta = opts->dmse_delta;
    net->stream = (hipStream_t)opts->hip_stream;
    const bool hbm = (opts->flags & SNN_FLAG_HBM_RINGS) != 0;

    int so = 0;
    for (int l = 0; l < n_layers; ++l) {
        t.n[l] = layers[l].n;
        t.kind[l] = layers[l].kind;
        t.lif[l] = -1;
        t.lif_off[l] = 0;
        t.bring[l] = -1;
        net->st_off[l] = so;
        if (l > 0) {
            so += layers[l].n;
            t.maxn = std::max(t.maxn, layers[l].n);
        }
        if (layers[l].kind == SNN_LIF) {
            t.lif[l] = t.n_lif++;
            t.lif_off[l] = t.lif_total;
            t.lif_total += layers[l].n;
        }
    }
    net->n_state = so;
    t.out_l = n_layers - 1;
    t.out_lif = dmse ? 1 : 0;
    long long off = 0;
    for (int l = 1; l < n_layers; ++l) {
        for (int r = 0; r < 1 + (layers[l].recurrent ? 1 : 0); ++r) {
            const int p = t.P++;
            t.pre[p] = r ? l : l - 1;
            t.post[p] = l;
            t.woff[p] = off;
            t.fring[p] = -1;
            net->cnt[p] = (long long)t.n[t.pre[p]] * t.n[l];
            off += net->cnt[p];
        }
    }
    net->n_params = off;
    t.out_p = t.P - 1;
    const int C = t.n[t.out_l];
    // delay rings as deep as each projection's largest delay
    for (int p = 0; p < t.P; ++p) {
        const int dm = opts->proj_max_delay ? opts->proj_max_delay[p] : max_delay;
        if (dm < 0 || dm > max_delay) {
            snprintf(g_create_err, sizeof(g_create_err),
                     "snn_create: proj_max_delay[%d] = %d outside [0, max_delay = %d]", p, dm, max_delay);
            free(net);
            return SNN_EINVAL;
        }
        t.dmax[p] = dm;
        t.Sp[p] = dm + 1;
    }
    // spike-count regulariser strengths, one per LIF layer
    for (int li = 0; li < t.n_lif && opts->reg_strength; ++li) {
        const float r = opts->reg_strength[li];
        if (!(r >= 0.0f) || isinf(r)) {
            snprintf(g_create_err, sizeof(g_create_err),
                     "snn_create: reg_strength[%d] must be finite and >= 0", li);
            free(net);
            return SNN_EINVAL;
        }
        net->reg_rho[li] = (double)r;
        if (r > 0.0f) net->reg_on = 1;
    }
    net->reg_nu = (double)opts->reg_target;
    for (int l = 0; l < n_layers; ++l) t.Sb[l] = 0;
    for (int p = 0; p < t.P; ++p)
        if (t.pre[p] != 0 && t.kind[t.post[p]] == SNN_LIF)
            t.Sb[t.post[p]] = std::max(t.Sb[t.post[p]], t.Sp[p]);

    // ---- LDS plans (the kernels' LDS limits first: occupancy depends on them)
    {
        int bad = -1;
        const char* what = "forward LDS limits";
        hipError_t e = set_forward_lds_limits(kLds, &bad);
        if (e == hipSuccess) {
            what = "forward core LDS limits";
            e = set_core_lds_limits(kLds, &bad);
        }
        if (e == hipSuccess) {
            what = "backward LDS limits";
            e = set_backward_lds_limits(kLds, &bad);
        }
        if (e != hipSuccess) {
            snprintf(g_create_err, sizeof(g_create_err), "snn_create: %s (kernel %d): %s", what, bad,
                     hipGetErrorString(e));
            free(net);
            return SNN_EDEVICE;
        }
    }
    int maxlif = 0;
    for (int l = 1; l < n_layers; ++l)
        if (t.kind[l] == SNN_LIF) maxlif = std::max(maxlif, t.n[l]);
    net->core_threads = std::max(64, ((maxlif + 63) / 64) * 64);
    const int nwaves = net->core_threads / 64;
    // cluster mode: CUs and cooperative launch support, LIF-post projections
    const bool want_cl = !hbm && t.n_lif > 0;
    const bool force_cl = (opts->flags & SNN_FLAG_CLUSTER) != 0;
    int n_cu = 256, coop = 0;
    {
        int dev = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            n_cu < 1)
            n_cu = 256;
        if (hipDeviceGetAttribute(&coop, hipDeviceAttributeCooperativeLaunch, dev) != hipSuccess) coop = 0;
    }
    net->cl_G = (maxlif + 63) / 64;
    for (int l = 1; l < n_layers; ++l) {
        if (t.kind[l] != SNN_LIF) continue;
        int k = 0;
        for (int p = 0; p < t.P; ++p)
            if (t.pre[p] == l && t.kind[t.post[p]] == SNN_LIF) ++k;
        net->cl_np = std::max(net->cl_np, k);
    }
    // forward core: the delay rings [S+1][n_post] of the LIF->LIF projections
    // (row S: dummy), all in LDS or all in HBM, then the ballot masks [3][NL][NW]
    {
        const size_t masks = align16((size_t)3 * std::max(t.n_lif, 1) * nwaves * sizeof(unsigned long long)) +
                             align16((size_t)std::max(t.n_lif, 1) * net->core_threads * sizeof(int));
        size_t used = 0;
        for (int p = 0; p < t.P; ++p) {
            if (t.pre[p] == 0 || t.kind[t.post[p]] != SNN_LIF) continue;
            t.fring[p] = (int)(used / sizeof(float));
            used += (size_t)(t.Sp[p] + 1) * t.n[t.post[p]] * sizeof(float);
        }
        const bool rings_lds = !(hbm || used + masks > kLds);
        if (!rings_lds) {
            used = 0;
            for (int p = 0; p < t.P; ++p) t.fring[p] = -1;
        }
        net->mask_off = (int)align16(used);
        net->ids_off = net->mask_off +
                       (int)align16((size_t)3 * std::max(t.n_lif, 1) * nwaves * sizeof(unsigned long long));
        net->lds_core_f = net->mask_off + masks;
        // cluster mode where the rings do not fit (or on request): each
        // workgroup holds 64 columns of every ring, the masks of all G
        // workgroups [3][NL][G] and an abort flag
        if (want_cl && coop && net->cl_np > 0 && (force_cl || !rings_lds)) {
            const int G = net->cl_G;
            size_t u = 0;
            int off[SNN_MAXP], rings = 0;
            for (int p = 0; p < t.P; ++p) {
                off[p] = -1;
                if (t.pre[p] == 0 || t.kind[t.post[p]] != SNN_LIF) continue;
                off[p] = (int)(u / sizeof(float));
                u += (size_t)(t.Sp[p] + 1) * 64 * sizeof(float);
                ++rings;
            }
            const size_t mk = align16((size_t)3 * t.n_lif * G * sizeof(unsigned long long)) + 16;
            const size_t lds = align16(u) + mk;
            const int threads = 64 * (1 + rings);
            int nb = 0;
            if (lds <= kLds &&
                forward_cluster_occupancy(t.n_lif, net->cl_np, threads, lds, &nb) == hipSuccess &&
                nb > 0 && (long long)n_cu * nb >= G) {
                net->cl_threads = threads;
                net->cl_f = 1;
                net->cl_spp_f = std::min<long long>((long long)n_cu * nb / G, t.B);
                for (int p = 0; p < t.P; ++p) t.fring[p] = off[p];
                net->mask_off = (int)align16(u);
                net->lds_core_f = lds;
            }
        }
        // the LI readout fed by a LIF layer as one more wave of the core: its
        // arrival ring [S_out + 1][C] after the masks
        const int feed_l = t.pre[t.out_p];
        const size_t ro_ring = (size_t)(t.Sp[t.out_p] + 1) * C * sizeof(float);
        if (!t.out_lif && feed_l != 0 && net->core_threads <= 256 && C <= 64 && !net->cl_f &&
            !(opts->flags & SNN_FLAG_SEPARATE_READOUT) &&
            align16(net->lds_core_f) + ro_ring <= kLds) {
            net->ro_fused = 1;
            net->ro_off = (int)align16(net->lds_core_f);
            net->lds_core_f = net->ro_off + ro_ring;
        }
    }
    // backward core: partial jump sums [2][NL][KP][4 NW] and the fp64 adjoint
    // rings [Sb][n] of the LIF layers read by LIF-pre projections (all in
    // LDS, or all in HBM)
    bool read_by_lif[SNN_MAX_LAYERS] = {false};
    for (int p = 0; p < t.P; ++p)
        if (t.pre[p] != 0 && t.kind[t.post[p]] == SNN_LIF) read_by_lif[t.post[p]] = true;
    {
        const int NL = std::max(t.n_lif, 1);
        const int KP = bwd_prefetch(NL);
        net->bpart_off = 0;
        const size_t part = align16((size_t)2 * NL * KP * 4 * nwaves * sizeof(double));
        size_t used = part;
        bool all_lds = !hbm;
        for (int l = 0; l < n_layers; ++l) {
            net->bring_mode[l] = -2;
            if (!read_by_lif[l]) continue;
            const size_t bytes = align16((size_t)t.Sb[l] * t.n[l] * sizeof(double));
            net->bring_mode[l] = (int)used;
            used += bytes;
        }
        if (used > kLds) all_lds = false;
        if (!all_lds) {
            used = part;
            for (int l = 0; l < n_layers; ++l)
                if (net->bring_mode[l] >= 0) net->bring_mode[l] = -1;
        }
        // cluster mode where the rings do not fit (or on request): the
        // exchange staging (shares [NL NP][KC][4], slot totals [NL KC],
        // own positions [NL][64], a flag), then 64 columns of every adjoint ring
        if (want_cl && coop && net->cl_np > 0 && (force_cl || !all_lds)) {
            const size_t stage = align16((size_t)NL * net->cl_np * kClKC * 4 * sizeof(double) +
                                         (size_t)NL * kClKC * sizeof(double) + (size_t)NL * 64 * sizeof(int) +
                                         sizeof(int));
            int rings = 0;
            for (int p = 0; p < t.P; ++p)
                if (t.pre[p] != 0 && t.kind[t.post[p]] == SNN_LIF) ++rings;
            const int threads = 64 * (1 + rings);
            size_t u = stage;
            int mode[SNN_MAX_LAYERS];
            for (int l = 0; l < n_layers; ++l) {
                mode[l] = -2;
                if (!read_by_lif[l]) continue;
                mode[l] = (int)u;
                u += align16((size_t)t.Sb[l] * 64 * sizeof(double));
            }
            int nb = 0;
            if (u <= kLds && backward_cluster_occupancy(NL, net->cl_np, threads, u, &nb) == hipSuccess &&
                nb > 0 && (long long)n_cu * nb >= net->cl_G) {
                net->cl_b = 1;
                net->cl_threads = threads;
                net->cl_spp_b = std::min<long long>((long long)n_cu * nb / net->cl_G, t.B);
                net->cl_off_b = 0;
                for (int l = 0; l < n_layers; ++l) net->bring_mode[l] = mode[l];
                used = u;
            }
        }
        for (int l = 0; l < n_layers; ++l) t.bring[l] = net->bring_mode[l] >= 0 ? net->bring_mode[l] : -1;
        net->lds_core_b = used;
    }
    // input scan: windows of 128 arrival steps (a [128][64] table per wave)
    // input scan ring: S + TB - 1 arrival steps and a dummy row per 64-post
    // wave; TB as large as keeps four rings in one CU's LDS (40 KiB each),
    // at least 8
    net->scan_tb = std::max(8, std::min(64, 160 - t.Sp[0]));
    net->lds_scan = (size_t)(t.Sp[0] + net->scan_tb) * 64 * sizeof(float);
    // readout forward: arrival table [T + 1][C] (row T: dummy) in LDS when it fits
    // readout: groups of ceil(C / 64) waves, each building a window of the
    // arrival table; up to 1024 threads
    {
        const int ob = (C + 63) / 64;
        net->read_threads = 64 * ob * std::max(1, 16 / ob);
    }
    {
        const size_t tab = align16((size_t)(t.T + 1) * C * sizeof(float));
        if (!hbm && tab <= kLds) {
            net->table_lds = 0;
            net->lds_read = tab;
        } else {
            net->table_lds = -1;
            net->lds_read = 0;
        }
    }
    // readout adjoint: the [T][C] table of lambda_I - lambda_V (fp64) in LDS when it fits
    net->radj_threads = 512;
    net->radj_tab = (!hbm && (size_t)t.T * C * sizeof(double) <= kLds) ? 1 : 0;
    net->lds_radj = net->radj_tab ? (size_t)t.T * C * sizeof(double) : 0;
    // gradients: one group per post layer (its projections in projection
    // order), J posts per workgroup, samples split into SB blocks so that the
    // grid has about 512 workgroups; workgroups in units of 4 J-blocks.  LDS:
    // the J trajectories of a sample [T + 1][J] double2 (row T: zeros), J =
    // 8, 4 or 2 (longer trials: J = 8 in windows of at most 1024 steps); the
    // spike-list offsets of the sample's presynaptic layers; the rest for its
    // spike steps (16-bit)
    const size_t grad_total = kLds;
    int grad_maxpre = 64;
    for (int q = 1; q < n_layers; ++q) {
        int v = 0;
        for (int p = 0; p < t.P; ++p)
            if (t.post[p] == q) v += t.n[t.pre[p]];
        grad_maxpre = std::max(grad_maxpre, v);
    }
    // the spike-list offsets of both presynaptic layers of a group
    const int grad_glcap = (grad_maxpre + 2 + 3) & ~3;
    {
        // the trajectories within 128 KiB, and within what the offsets and
        // 16 KiB of spike steps leave
        const size_t tb = std::min<size_t>(128 * 1024, grad_total - (size_t)grad_glcap * sizeof(int) - 16 * 1024);
        const size_t tj = ((size_t)t.T + 1) * sizeof(double2);
        net->grad_J = 0;
        net->grad_TW = t.T;
        for (int j : {8, 4, 2})
            if (!net->grad_J && j * tj <= tb) net->grad_J = j;
        if (!net->grad_J) {
            net->grad_J = 8;
            net->grad_TW = std::min(1024, (int)(tb / (8 * sizeof(double2))) - 1);
        }
        const int J = net->grad_J;
        int ng = 0, jblocks = 0, maxpre = 64;
        for (int q = 1; q < n_layers; ++q) {
            GradGroup& g = net->grad_grp[ng];
            g = GradGroup{};
            g.nq = t.n[q];
            g.jb = (g.nq + J - 1) / J;
            g.out = (q == t.out_l && !t.out_lif) ? 1 : 0;
            g.off = g.out ? 0 : t.lif_off[q];
            for (int p = 0; p < t.P; ++p) {
                if (t.post[p] != q) continue;
                g.p[g.np] = p;
                g.pre[g.np] = t.pre[p];
                g.npre[g.np] = t.n[t.pre[p]];
                ++g.np;
            }
            maxpre = std::max(maxpre, g.npre[0] + (g.np > 1 ? g.npre[1] : 0));
            jblocks += g.jb;
            ++ng;
        }
        // sample blocks: a workgroup holds a CU (its LDS), so the grid runs in
        // rounds of n_cu workgroups; take the SB that minimises rounds x
        // samples per block (the fp64 partials of SB > 1 blocks capped at
        // 512 MiB)
        int n_cu = 256, dev = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            n_cu < 1)
            n_cu = 256;
        const long long part_cap = (512ll << 20) / (16ll * std::max<long long>(net->n_params, 1));
        auto cost_of = [&](int sb) {
            const int bsz = (t.B + sb - 1) / sb;
            return (((long long)jblocks * sb + n_cu - 1) / n_cu) * bsz;
        };
        long long best = -1;
        for (int sb = 1; sb <= t.B && (sb == 1 || sb <= part_cap); ++sb) {
            const long long c = cost_of(sb);
            if (best < 0 || c < best) best = c;
        }
        // the fewest blocks (least partial-sum traffic) within 3 % of it
        int SB = 1;
        while (SB < t.B && cost_of(SB) * 100 > best * 103) ++SB;
        const int bs = (t.B + SB - 1) / SB;
        SB = (t.B + bs - 1) / bs;                            // no empty trailing block
        int blk = 0;
        for (int g = 0; g < ng; ++g) {
            GradGroup& G = net->grad_grp[g];
            G.blk0 = blk;
            G.units = (((G.jb + 3) / 4) * SB + 7) / 8 * 8;
            blk += G.units * 4;
        }
        net->grad_ngroups = ng;
        net->grad_SB = SB;
        net->grad_bs = bs;
        net->grad_nblk = blk;
        // synapses of a block: J x maxpre, dealt KL per lane (one pass when they fit)
        const int pairs = J * maxpre;
        net->grad_KL = (pairs <= 4 * 1024) ? 4 : 8;
        net->grad_threads = std::min(1024, ((pairs + net->grad_KL - 1) / net->grad_KL + 63) / 64 * 64);
        const size_t traj = (size_t)J * (net->grad_TW + 1) * sizeof(double2);
        const size_t gl = (size_t)grad_glcap * sizeof(int);
        const size_t room = (traj + gl < grad_total) ? grad_total - traj - gl : 0;
        // (eight entries of slack: a spike loop reads up to three past a list)
        const size_t ent = room / sizeof(unsigned short);
        net->grad_spcap = (int)(ent >= 8 ? ent - 8 : 0) & ~7;
        net->grad_glcap = grad_glcap;
        net->lds_grad = traj + gl + (size_t)(net->grad_spcap + 8) * sizeof(unsigned short);
    }

    // ---- device scratch
    hipError_t e = hipSuccess;
    const size_t B = t.B, T = (size_t)t.T, T1 = T + 1, cap = (size_t)t.cap;
    const size_t nl = (size_t)std::max(t.n_lif, 1);
    const int feed = t.pre[t.out_p];
#define ALLOC(ptr, count)                                 \
    if (e == hipSuccess) e = dalloc(&(ptr), (count));
    ALLOC(net->slot, (size_t)net->n_params);
    ALLOC(net->ws, (size_t)net->n_params);
    ALLOC(net->steptab, nl * B * T * (size_t)SNN_STEP_ROW);
    ALLOC(net->in_idx, B * T1);
    ALLOC(net->A_in, B * T * t.n[1]);
    for (int p = 0; p < t.P; ++p)
        if (t.pre[p] != 0 && t.kind[t.post[p]] == SNN_LIF && t.fring[p] < 0)
            ALLOC(net->fring[p], B * (t.Sp[p] + 1) * t.n[t.post[p]]);
    for (int l = 1; l < n_layers; ++l)
        if (net->bring_mode[l] == -1) ALLOC(net->bring[l], B * t.Sb[l] * t.n[l]);
    ALLOC(net->rec_n, nl * B * cap);
    ALLOC(net->rec_s, nl * B * cap);
    ALLOC(net->rec_I, nl * B * cap);
    ALLOC(net->rec_idx, nl * B * T1);
    ALLOC(net->rec_cnt, nl * B);
    ALLOC(net->rec_goff, nl * B * (t.maxn + 1));
    // (per layer a multiple of 8 entries, so that every layer starts 16-byte
    // aligned, and slack: the gradient pass copies the 16-bit lists as dwords)
    ALLOC(net->rec_gstep, nl * gstep_stride(B, cap) + 8);
    ALLOC(net->z, B * C);
    ALLOC(net->nstar, B * C);
    ALLOC(net->src, B * C);
    ALLOC(net->Vf, B * so);
    ALLOC(net->If, B * so);
    if (net->table_lds < 0) ALLOC(net->table, B * (T + 1) * C);
    ALLOC(net->tr_lif, B * T * t.lif_total);
    ALLOC(net->tr_out, B * T * C);
    if (net->grad_SB > 1) ALLOC(net->gpart, (size_t)net->grad_SB * 2 * (size_t)net->n_params);
    if (feed != 0 && !t.out_lif) ALLOC(net->A2, B * cap);
    if (t.out_lif) ALLOC(net->xlp_out, B * cap);
    if (net->reg_on) {
        ALLOC(net->ncount, (size_t)t.lif_total);
        ALLOC(net->nterm, (size_t)t.lif_total);
        // summed jump terms of the regularised layers (the layer feeding an
        // LI readout adds them into its readout part in place)
        for (int l = 1; l < n_layers; ++l) {
            if (t.kind[l] != SNN_LIF || net->reg_rho[t.lif[l]] == 0.0) continue;
            if (!(!t.out_lif && l == feed)) ALLOC(net->jx[t.lif[l]], B * cap);
        }
    }
    ALLOC(net->in_goff, B * (t.n_in + 1));
    ALLOC(net->st, 1);
    if (net->cl_f || net->cl_b) {
        // exchange words of every cluster slot, two parities (zero: no tag)
        const size_t fw = net->cl_f ? (size_t)net->cl_spp_f * 2 * nl * net->cl_G : 0;
        const size_t bw = net->cl_b ? (size_t)net->cl_spp_b * net->cl_G * 2 * nl * kClKC : 0;
        const size_t words = 2 * std::max(fw, bw);
        ALLOC(net->clx, words);
        if (e == hipSuccess) e = hipMemset(net->clx, 0, words * sizeof(unsigned long long));
        net->cl_tag = 1;
    }
#undef ALLOC
    const char* what = "device allocation";
    int bad = -1;   // index of the kernel whose LDS limit was refused
    if (e == hipSuccess) e = hipHostMalloc((void**)&net->st_host, sizeof(DevStatus), hipHostMallocDefault);
    if (e == hipSuccess) {
        what = "scratch symbol address";
        e = scratch_address(&net->scratch);
    }
    if (e == hipSuccess) {
        what = "auxiliary stream";
        e = hipStreamCreateWithFlags(&net->aux, hipStreamNonBlocking);
    }
    if (e == hipSuccess) e = hipEventCreateWithFlags(&net->fork, hipEventDisableTiming);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&net->join, hipEventDisableTiming);
    net->timing = (opts->flags & SNN_FLAG_TIMING) ? 1 : 0;
    if (e == hipSuccess) what = "timing events";
    for (int i = 0; i < 2 * K_N && net->timing && e == hipSuccess; ++i) e = hipEventCreate(&net->ev[i]);
    if (e != hipSuccess) {
        snprintf(g_create_err, sizeof(g_create_err), "snn_create: %s (kernel %d): %s", what, bad,
                 hipGetErrorString(e));
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

#define TIMED(net, k, expr)                                                                 \
    do {                                                                                    \
        (net)->ran[k] = 1;                                                                  \
        if ((net)->timing) HIP_TRY(net, hipEventRecord((net)->ev[2 * (k)], (net)->stream)); \
        HIP_TRY(net, expr);                                                                 \
        if ((net)->timing)                                                                  \
            HIP_TRY(net, hipEventRecord((net)->ev[2 * (k) + 1], (net)->stream));           \
    } while (0)

static int collect_times(snn_net* net, int k0, int k1) {
    if (!net->timing) return SNN_OK;
    for (int k = k0; k < k1; ++k) {
        net->stats.kernel_ms[k] = 0.0f;
        if (!net->ran[k]) continue;
        HIP_TRY(net, hipEventElapsedTime(&net->stats.kernel_ms[k], net->ev[2 * k], net->ev[2 * k + 1]));
    }
    return SNN_OK;
}

// The cluster-mode cores: one cooperative launch per pass of cl_spp samples,
// each with tags of its own (the tag advances by 2 per exchange: one per
// step forward, at most ceil(widest layer / KP) per step backward).
static hipError_t launch_forward_clusters(snn_net* net, CoreFwdArgs& a, hipStream_t s) {
    const Topo& t = net->t;
    a.NW = net->cl_G;
    a.ro_C = 0;
    a.cl.G = net->cl_G;
    a.cl.x = net->clx;
    for (int b0 = 0; b0 < t.B; b0 += net->cl_spp_f) {
        const int nc = std::min(net->cl_spp_f, t.B - b0);
        a.cl.b0 = b0;
        a.cl.tag0 = net->cl_tag;
        net->cl_tag += 2u * (unsigned)t.T;
        const hipError_t e = launch_forward_core_cluster(a, t.n_lif, net->cl_np, nc * net->cl_G,
                                                         net->cl_threads, net->lds_core_f, s);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

static hipError_t launch_backward_clusters(snn_net* net, CoreBwdArgs& a, hipStream_t s) {
    const Topo& t = net->t;
    a.NW = 1;
    a.cl.G = net->cl_G;
    a.cl.x = net->clx;
    a.cl_off = net->cl_off_b;
    hipError_t e = launch_clear_abort(net->st, s);
    for (int b0 = 0; b0 < t.B && e == hipSuccess; b0 += net->cl_spp_b) {
        const int nc = std::min(net->cl_spp_b, t.B - b0);
        a.cl.b0 = b0;
        a.cl.tag0 = net->cl_tag;
        net->cl_tag += 2u * ((unsigned)t.T * (unsigned)((t.maxn + kClKC - 1) / kClKC) + 1u);
        e = launch_backward_core_cluster(a, t.n_lif, net->cl_np, nc * net->cl_G, net->cl_threads,
                                         net->lds_core_b, s);
    }
    return e;
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
    const int C = t.n[t.out_l];
    for (int k = K_SCAN; k < K_RADJ; ++k) net->ran[k] = 0;
    HIP_TRY(net, launch_reset_status(net->st, s));
    HIP_TRY(net, launch_validate(in->offsets, in->step, in->neuron, in->nnz, t.B, t.T, t.n_in, labels,
                                 C, net->st, s));
    HIP_TRY(net, launch_step_index(in->offsets, in->step, t.B, t.T, net->in_idx, net->st, s));
    HIP_TRY(net, launch_round_delays(D, W, t.woff, net->cnt, t.P, t.dmax, net->slot, net->ws,
                                     net->st, s));

    InScanArgs sa{};
    sa.B = t.B;
    sa.T = t.T;
    sa.S = t.Sp[0];
    sa.n_in = t.n_in;
    sa.n1 = t.n[1];
    sa.TB = net->scan_tb;
    sa.ws0 = net->ws;
    sa.in_neuron = in->neuron;
    sa.in_step = in->step;
    sa.in_idx = net->in_idx;
    sa.A_in = net->A_in;
    sa.st = net->st;
    TIMED(net, K_SCAN, launch_input_scan(sa, net->lds_scan, s));

    if (net->reg_on) HIP_TRY(net, launch_zero_ints(net->ncount, t.lif_total, s));
    if (t.n_lif > 0) {
        CoreFwdArgs a{};
        a.B = t.B;
        a.T = t.T;
        a.cap = t.cap;
        a.NW = net->core_threads / 64;
        a.n1 = t.n[1];
        a.nstate = net->n_state;
        a.alpha = t.alpha;
        a.beta = t.beta;
        a.gamma = t.gamma;
        a.theta = t.theta;
        const size_t B = t.B, cap = t.cap;
        for (int l = 1; l < t.L; ++l) {
            if (t.kind[l] != SNN_LIF) continue;
            const int li = t.lif[l];
            FwdLayer& y = a.ly[li];
            y.n = t.n[l];
            a.soff[li] = net->st_off[l];
            // projections into the layer, in projection order
            for (int p = 0; p < t.P; ++p) {
                if (t.post[p] != l) continue;
                const int pre = t.pre[p];
                y.in_l[y.nin] = (pre == 0) ? -1 : t.lif[pre];
                y.in_pp[y.nin] = 0;
                y.in_S[y.nin] = t.Sp[p];
                y.in_ring_lds[y.nin] = t.fring[p];
                y.in_ring[y.nin] = net->fring[p];
                if (pre != 0) {
                    // position of p among the LIF-post projections of its source layer
                    int k = 0;
                    for (int p2 = 0; p2 < p; ++p2)
                        if (t.pre[p2] == pre && t.kind[t.post[p2]] == SNN_LIF) ++k;
                    y.in_pp[y.nin] = k;
                }
                ++y.nin;
            }
            // LIF-post projections out of the layer, in projection order
            for (int p = 0; p < t.P; ++p) {
                const int q = t.post[p];
                if (t.pre[p] != l || t.kind[q] != SNN_LIF) continue;
                y.nq[y.npost] = t.n[q];
                y.npre[y.npost] = t.n[l];
                y.S[y.npost] = t.Sp[p];
                y.ring_lds[y.npost] = t.fring[p];
                y.ring[y.npost] = net->fring[p];
                y.ws[y.npost] = net->ws + t.woff[p];
                ++y.npost;
            }
            for (int k = y.npost; k < 2; ++k) {
                // any LIF-post projection of the network stands in for unused entries
                for (int p = 0; p < t.P && !y.ws[k]; ++p) {
                    const int q = t.post[p];
                    if (t.pre[p] == 0 || t.kind[q] != SNN_LIF) continue;
                    y.nq[k] = t.n[q];
                    y.npre[k] = t.n[t.pre[p]];
                    y.S[k] = t.Sp[p];
                    y.ring_lds[k] = t.fring[p];
                    y.ring[k] = net->fring[p];
                    y.ws[k] = net->ws + t.woff[p];
                }
            }
            y.rec_n = net->rec_n + li * B * cap;
            y.rec_s = net->rec_s + li * B * cap;
            y.rec_I = net->rec_I + li * B * cap;
            y.rec_idx = net->rec_idx + li * B * (size_t)(t.T + 1);
            y.rec_cnt = net->rec_cnt + li * B;
            y.steptab = net->steptab + li * B * (size_t)t.T * SNN_STEP_ROW;
            y.ncount = net->reg_on ? net->ncount + t.lif_off[l] : nullptr;
            y.out_count = records[li].count;
            y.out_step = records[li].step;
            y.out_neuron = records[li].neuron;
        }
        a.A_in = net->A_in;
        a.Vf = net->Vf;
        a.If = net->If;
        a.st = net->st;
        a.mask_off = net->mask_off;
        a.ids_off = net->ids_off;
        if (net->ro_fused) {
            a.ro_C = C;
            a.ro_feed = t.lif[t.pre[t.out_p]];
            a.ro_nfeed = t.n[t.pre[t.out_p]];
            a.ro_S = t.Sp[t.out_p];
            a.ro_off = net->ro_off;
            a.ro_loss = t.loss;
            a.ro_scale = t.rscale;
            a.ro_ws = net->ws + t.woff[t.out_p];
            a.z = net->z;
            a.nstar = net->nstar;
        }
        if (net->cl_f)
            TIMED(net, K_CORE, launch_forward_clusters(net, a, s));
        else
            TIMED(net, K_CORE, launch_forward_core(a, t.n_lif, net->core_threads + (net->ro_fused ? 64 : 0),
                                                   net->lds_core_f, s));
    }
    if (net->reg_on) {
        RegArgs ra{};
        ra.nl = t.n_lif;
        ra.B = t.B;
        ra.nu = net->reg_nu;
        ra.st = net->st;
        for (int l = 1; l < t.L; ++l) {
            if (t.kind[l] != SNN_LIF) continue;
            const int li = t.lif[l];
            ra.n[li] = t.n[l];
            ra.rho[li] = net->reg_rho[li];
            ra.ncount[li] = net->ncount + t.lif_off[l];
            ra.nterm[li] = net->nterm + t.lif_off[l];
        }
        HIP_TRY(net, launch_spike_reg(ra, s));
    }
    if (t.out_lif) {
        // spike-time loss on the first spikes of the LIF output layer
        const size_t li = (size_t)t.lif[t.out_l], B = t.B, cap = t.cap;
        HIP_TRY(net, launch_dmse_loss(net->rec_cnt + li * B, net->rec_s + li * B * cap,
                                      net->rec_n + li * B * cap, t.cap, labels, t.B, C, t.T, t.dt,
                                      net->dmse_delta, net->z, loss, net->xlp_out, net->st, s));
    } else {
        if (!net->ro_fused) {
            ReadoutArgs r{};
            r.t = t;
            r.ws = net->ws + t.woff[t.out_p];
            r.A_in = net->A_in;
            r.rec_n = net->rec_n;
            r.rec_s = net->rec_s;
            r.rec_idx = net->rec_idx;
            r.table = net->table;
            r.table_lds = net->table_lds;
            r.z = net->z;
            r.nstar = net->nstar;
            r.Vf = net->Vf;
            r.If = net->If;
            r.st = net->st;
            TIMED(net, K_READ, launch_readout_forward(r, net->read_threads, net->lds_read, s));
        }
        HIP_TRY(net, launch_loss(net->z, labels, t.B, C, t.loss, t.rscale, net->tau_m, loss,
                                 net->src, net->st, s));
    }
    if (z)
        HIP_TRY(net, hipMemcpyAsync(z, net->z, sizeof(float) * t.B * C, hipMemcpyDeviceToDevice, s));
    int rc = read_status(net);
    if (rc) return rc;
    const DevStatus& h = *net->st_host;
    if (h.bad_input)
        return fail(net, SNN_EINVAL, "input spikes or labels invalid (offsets, range, order)");
    if (h.cl_abort)
        return fail(net, SNN_EDEVICE, "forward core: a cluster exchange timed out (results void)");
    memset(&net->stats, 0, sizeof(net->stats));
    rc = collect_times(net, K_SCAN, K_RADJ);
    if (rc) return rc;
    net->stats.input_spikes = in->nnz;
    net->stats.clamped_delays = (int64_t)h.clamped;
    net->stats.reg_loss = h.reg_loss;
    net->stats.overflow = h.overflow;
    for (int p = 0; p < t.P; ++p)
        if (t.fring[p] >= 0) net->stats.lds_rings |= 1 << p;
    long long ev = 0;
    for (int p = 0; p < t.P; ++p) {
        const int pre = t.pre[p];
        const long long spikes = (pre == 0) ? in->nnz : (long long)h.layer_spikes[t.lif[pre]];
        ev += spikes * t.n[t.post[p]];
    }
    for (int li = 0; li < t.n_lif; ++li) net->stats.lif_spikes += (int64_t)h.layer_spikes[li];
    net->stats.events = ev;
    for (int p = 0; p < t.P; ++p) net->W[p] = W[p];
    net->in_off = in->offsets;
    net->in_step = in->step;
    net->in_neuron = in->neuron;
    net->in_nnz = in->nnz;
    net->fwd_ok = 1;
    net->fwd_overflow = h.overflow;
    if (h.overflow) return fail(net, SNN_EOVERFLOW, "a sample exceeded record_capacity spikes");
    return SNN_OK;
}

// The backward pass.  in_goff / in_gstep: where the input spikes grouped by
// channel go ([B][n_in + 1] int32 and [nnz + 8] 16-bit); NULL: the handle's own buffers
// (in_gstep grown on demand).
static int backward_impl(snn_net* net, const float* const* dlp, float* const* dW, float* const* dD,
                         int* in_goff, unsigned short* in_gstep) {
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
    for (int k = K_RADJ; k < K_N; ++k) net->ran[k] = 0;
    // per-record jump terms from the caller on a LIF layer: device room for
    // their fp64 sums (first use of the layer)
    bool has_lp[SNN_MAX_LIF] = {false};
    for (int li = 0; dlp && li < t.n_lif; ++li) {
        if (!dlp[li] || t.cap < 1) continue;
        has_lp[li] = true;
        if (net->jx[li]) continue;
        const hipError_t e = hipMalloc((void**)&net->jx[li], (size_t)t.B * t.cap * sizeof(double));
        if (e != hipSuccess) {
            net->jx[li] = nullptr;
            return fail(net, e == hipErrorOutOfMemory ? SNN_ENOMEM : SNN_EDEVICE, "hipMalloc: %s",
                        hipGetErrorString(e));
        }
    }
    // the grouped input steps need one slot per input spike of the last forward
    if (!in_gstep && net->in_nnz > net->in_gstep_cap) {
        HIP_TRY(net, hipStreamSynchronize(s));
        if (net->in_gstep) HIP_TRY(net, hipFree(net->in_gstep));
        net->in_gstep = nullptr;
        net->in_gstep_cap = 0;
        const hipError_t e =
            hipMalloc((void**)&net->in_gstep, ((size_t)net->in_nnz + 8) * sizeof(unsigned short));
        if (e != hipSuccess)
            return fail(net, e == hipErrorOutOfMemory ? SNN_ENOMEM : SNN_EDEVICE, "hipMalloc: %s",
                        hipGetErrorString(e));
        net->in_gstep_cap = net->in_nnz;
    }
    if (!in_goff) in_goff = net->in_goff;
    if (!in_gstep) in_gstep = net->in_gstep;
    const int C = t.n[t.out_l];
    const int feed = t.pre[t.out_p];
    const size_t B = t.B, cap = t.cap;
    if (!t.out_lif) {
        ReadoutBwdArgs r{};
        r.B = t.B;
        r.T = t.T;
        r.C = C;
        r.cap = t.cap;
        r.loss = t.loss;
        r.alpha = net->alpha64;
        r.beta = net->beta64;
        r.cc = net->cc64;
        // chunks of at least 8 steps, one lane per (output, chunk), and the
        // free propagator over a whole chunk
        {
            const int nch = std::max(1, std::min(net->radj_threads / C, (t.T + 7) / 8));
            r.LC = (t.T + nch - 1) / nch;
            r.nch = (t.T + r.LC - 1) / r.LC;
            double p11 = 1.0, p12 = 0.0, p22 = 1.0;
            for (int j = 0; j < r.LC; ++j) {
                p12 = r.beta * p12 + r.cc * p22;
                p11 = r.beta * p11;
                p22 = r.alpha * p22;
            }
            r.P11 = p11;
            r.P12 = p12;
            r.P22 = p22;
        }
        r.ws = net->ws + t.woff[t.out_p];
        if (feed != 0) {
            const size_t li = (size_t)t.lif[feed];
            r.rec_n = net->rec_n + li * B * cap;
            r.rec_s = net->rec_s + li * B * cap;
            r.rec_cnt = net->rec_cnt + li * B;
        }
        r.nstar = net->nstar;
        r.src = net->src;
        r.traj = net->tr_out;
        r.A2 = net->A2;
        r.tab_lds = net->radj_tab;
        TIMED(net, K_RADJ, launch_readout_adjoint(r, net->radj_threads, net->lds_radj, s));
    }
    // spikes grouped by presynaptic neuron (inputs, then every LIF layer) on
    // the second stream: they depend on the forward only, and run beside the
    // latency-bound adjoint core (forked after the readout adjoint, whose
    // workgroups take a whole CU's LDS); the gradients wait for them
    const hipStream_t g_s = net->aux;
    HIP_TRY(net, hipEventRecord(net->fork, s));
    HIP_TRY(net, hipStreamWaitEvent(g_s, net->fork, 0));
    net->ran[K_GROUP] = 1;
    if (net->timing) HIP_TRY(net, hipEventRecord(net->ev[2 * K_GROUP], g_s));
    {
        GroupArgs g{};
        g.off = net->in_off;
        g.end = net->in_off;
        g.step = net->in_step;
        g.neuron = net->in_neuron;
        g.n = t.n_in;
        g.g_off = in_goff;
        g.g_step = in_gstep;
        g.stage_cap = (int)std::min<long long>(net->in_nnz, kGroupStage);
        g.st = net->st;
        HIP_TRY(net, launch_group(g, t.B, g_s));
    }
    for (int l = 1; l < t.L; ++l) {
        if (t.kind[l] != SNN_LIF) continue;
        const size_t li = (size_t)t.lif[l];
        GroupArgs g{};
        g.cnt = net->rec_cnt + li * t.B;
        g.off_stride = t.cap;
        g.step = net->rec_s + li * t.B * t.cap;
        g.neuron = net->rec_n + li * t.B * t.cap;
        g.n = t.n[l];
        g.g_off = net->rec_goff + li * t.B * (t.maxn + 1);
        g.g_step = net->rec_gstep + li * gstep_stride(t.B, t.cap);
        g.stage_cap = std::min(t.cap, kGroupStage);
        g.st = net->st;
        HIP_TRY(net, launch_group(g, t.B, g_s));
    }
    if (net->timing) HIP_TRY(net, hipEventRecord(net->ev[2 * K_GROUP + 1], g_s));
    HIP_TRY(net, hipEventRecord(net->join, g_s));
    // extra jump numerators per LIF layer: the readout part of the jump sums
    // (the layer feeding an LI readout), the spike-time loss's terms (LIF
    // output layer), plus the caller's dl_p/dt
    const double* jump_x[SNN_MAX_LIF] = {nullptr};
    // and the spike-count regulariser's term of each record's neuron
    for (int l = 1; l < t.L; ++l) {
        if (t.kind[l] != SNN_LIF) continue;
        const int li = t.lif[l];
        const double* own = (!t.out_lif && l == feed) ? net->A2 : (t.out_lif && l == t.out_l) ? net->xlp_out : nullptr;
        const bool reg = net->reg_on && net->reg_rho[li] != 0.0;
        if (has_lp[li] || reg) {
            double* dst = (own == net->A2 && own) ? net->A2 : net->jx[li];
            HIP_TRY(net, launch_add_lp(dst, own, has_lp[li] ? dlp[li] : nullptr,
                                       reg ? net->nterm + t.lif_off[l] : nullptr,
                                       net->rec_n + (size_t)li * B * cap,
                                       net->rec_cnt + (size_t)li * B, t.B, t.cap, s));
            jump_x[li] = dst;
        } else {
            jump_x[li] = own;
        }
    }
    if (t.n_lif > 0) {
        CoreBwdArgs a{};
        a.B = t.B;
        a.T = t.T;
        a.cap = t.cap;
        a.NW = net->core_threads / 64;
        a.lif_total = t.lif_total;
        a.alpha = net->alpha64;
        a.beta = net->beta64;
        a.cc = net->cc64;
        a.theta = (double)t.theta;
        for (int l = 1; l < t.L; ++l) {
            if (t.kind[l] != SNN_LIF) continue;
            const size_t li = (size_t)t.lif[l];
            BwdLayer& y = a.ly[li];
            y.n = t.n[l];
            y.lif_off = t.lif_off[l];
            y.S = std::max(t.Sb[l], 1);
            y.ring_lds = net->bring_mode[l];
            y.ring = net->bring[l];
            for (int p = 0; p < t.P; ++p) {
                const int q = t.post[p];
                if (t.pre[p] != l || t.kind[q] != SNN_LIF) continue;
                y.ws[y.npost] = net->ws + t.woff[p];
                y.nq[y.npost] = t.n[q];
                y.npre[y.npost] = t.n[l];
                y.qS[y.npost] = t.Sb[q];
                y.qring_lds[y.npost] = net->bring_mode[q] >= 0 ? net->bring_mode[q] : -1;
                y.qring[y.npost] = net->bring[q];
                ++y.npost;
            }
            for (int k = y.npost; k < 2; ++k) {
                // any LIF-post projection of the network stands in for unused entries
                for (int p = 0; p < t.P && !y.ws[k]; ++p) {
                    const int q = t.post[p];
                    if (t.pre[p] == 0 || t.kind[q] != SNN_LIF) continue;
                    y.ws[k] = net->ws + t.woff[p];
                    y.nq[k] = t.n[q];
                    y.npre[k] = t.n[t.pre[p]];
                    y.qS[k] = t.Sb[q];
                    y.qring_lds[k] = net->bring_mode[q] >= 0 ? net->bring_mode[q] : -1;
                    y.qring[k] = net->bring[q];
                }
            }
            y.recI = net->rec_I + li * B * cap;
            y.recn = net->rec_n + li * B * cap;
            y.steptab = net->steptab + li * B * (size_t)t.T * SNN_STEP_ROW;
            y.A2 = jump_x[li];
        }
        a.traj = net->tr_lif;
        a.st = net->st;
        a.part_off = net->bpart_off;
        if (net->cl_b)
            TIMED(net, K_BCORE, launch_backward_clusters(net, a, s));
        else
            TIMED(net, K_BCORE,
                  launch_backward_core(a, t.n_lif, net->core_threads, net->lds_core_b, s));
    }
    HIP_TRY(net, hipStreamWaitEvent(s, net->join, 0));
    GradArgs ga{};
    ga.B = t.B;
    ga.T = t.T;
    ga.TW = net->grad_TW;
    ga.SB = net->grad_SB;
    ga.spcap = net->grad_spcap;
    ga.glcap = net->grad_glcap;
    ga.bs = net->grad_bs;
    ga.lif_total = t.lif_total;
    ga.C = C;
    ga.ngroups = net->grad_ngroups;
    ga.nblk = net->grad_nblk;
    ga.tau_s = t.tau_s;
    ga.dt = t.dt;
    ga.nparams = net->n_params;
    ga.tr_lif = net->tr_lif;
    ga.tr_out = net->tr_out;
    for (int p = 0; p < t.P; ++p) {
        ga.woff[p] = t.woff[p];
        ga.dW[p] = dW[p];
        ga.dD[p] = dD[p];
    }
    ga.ws = net->ws;
    ga.g_off[0] = in_goff;
    ga.g_step[0] = in_gstep;
    for (int l = 1; l < t.L; ++l) {
        if (t.kind[l] != SNN_LIF) continue;
        const size_t li = (size_t)t.lif[l];
        ga.g_off[l] = net->rec_goff + li * t.B * (t.maxn + 1);
        ga.g_step[l] = net->rec_gstep + li * gstep_stride(t.B, t.cap);
    }
    for (int g = 0; g < net->grad_ngroups; ++g) ga.grp[g] = net->grad_grp[g];
    ga.part = net->gpart;
    net->ran[K_GRAD] = 1;
    if (net->timing) HIP_TRY(net, hipEventRecord(net->ev[2 * K_GRAD], s));
    HIP_TRY(net, launch_gradients(ga, net->grad_J, net->grad_KL, net->grad_threads, net->lds_grad, s));
    if (ga.SB > 1) HIP_TRY(net, launch_grad_reduce(ga, t.P, s));
    if (net->timing) HIP_TRY(net, hipEventRecord(net->ev[2 * K_GRAD + 1], s));
    int rc = read_status(net);
    if (rc) return rc;
    if (net->st_host->cl_abort)
        return fail(net, SNN_EDEVICE, "backward core: a cluster exchange timed out (results void)");
    rc = collect_times(net, K_RADJ, K_N);
    if (rc) return rc;
    net->stats.degenerate_jumps = (int64_t)net->st_host->degenerate;
    return SNN_OK;
}

extern "C" int snn_backward(snn_net* net, float* const* dW, float* const* dD) {
    return backward_impl(net, nullptr, dW, dD, nullptr, nullptr);
}

extern "C" int snn_backward_lp(snn_net* net, const float* const* dlp, float* const* dW,
                               float* const* dD) {
    return backward_impl(net, dlp, dW, dD, nullptr, nullptr);
}

extern "C" int snn_backward_noalloc(snn_net* net, float* const* dW, float* const* dD) {
    if (!net) return SNN_EINVAL;
    const long long need = (long long)net->t.B * (net->t.n_in + 1) + net->in_nnz;
    if (need > kScratchInts)
        return fail(net, SNN_EINVAL,
                    "snn_backward_noalloc: the grouped input spikes need %lld int32, the fixed "
                    "scratch holds %lld (batch x (inputs + 1) + input spikes)",
                    need, (long long)kScratchInts);
    if (!net->scratch)
        return fail(net, SNN_EDEVICE, "snn_backward_noalloc: no scratch address for this device");
    int* goff = net->scratch;
    return backward_impl(net, nullptr, dW, dD, goff,
                         reinterpret_cast<unsigned short*>(goff + (size_t)net->t.B * (net->t.n_in + 1)));
}

extern "C" int snn_optimizer_step(snn_net* net, const snn_optim* o, float* const* W, float* const* D,
                                  const float* const* dW, const float* const* dD) {
    if (!net) return SNN_EINVAL;
    net->err[0] = 0;
    const Topo& t = net->t;
    if (!o || !W || !D || !dW || !dD) return fail(net, SNN_EINVAL, "NULL optimiser, W, D, dW or dD");
    if (o->kind != SNN_OPT_SGD && o->kind != SNN_OPT_ADAM)
        return fail(net, SNN_EINVAL, "unknown optimiser kind %d", o->kind);
    if (!(o->lr_w >= 0.0f) || !(o->lr_d >= 0.0f) || isinf(o->lr_w) || isinf(o->lr_d))
        return fail(net, SNN_EINVAL, "learning rates must be finite and >= 0");
    if (!(o->d_min <= o->d_max)) return fail(net, SNN_EINVAL, "d_min > d_max (or NaN)");
    if (o->kind == SNN_OPT_ADAM &&
        (!(o->beta1 >= 0.0f && o->beta1 < 1.0f) || !(o->beta2 >= 0.0f && o->beta2 < 1.0f) ||
         !(o->eps > 0.0f)))
        return fail(net, SNN_EINVAL, "Adam needs 0 <= beta1, beta2 < 1 and eps > 0");
    OptArgs a{};
    a.P = t.P;
    a.kind = o->kind;
    a.nparams = net->n_params;
    for (int p = 0; p < t.P; ++p) {
        if (!W[p] || !D[p] || !dW[p] || !dD[p])
            return fail(net, SNN_EINVAL, "NULL W, D, dW or dD of projection %d", p);
        const float sw = o->lr_scale_w ? o->lr_scale_w[p] : 1.0f;
        const float sd = o->lr_scale_d ? o->lr_scale_d[p] : 1.0f;
        if (!(sw >= 0.0f) || !(sd >= 0.0f) || isinf(sw) || isinf(sd))
            return fail(net, SNN_EINVAL, "learning-rate factors of projection %d must be finite and >= 0", p);
        a.woff[p] = t.woff[p];
        a.W[p] = W[p];
        a.D[p] = D[p];
        a.dW[p] = dW[p];
        a.dD[p] = dD[p];
        a.lr_w[p] = (float)((double)o->lr_w * sw);
        a.lr_d[p] = (float)((double)o->lr_d * sd);
    }
    a.d_min = o->d_min;
    a.d_max = o->d_max;
    if (o->kind == SNN_OPT_ADAM) {
        if (!net->mom) {
            const size_t bytes = (size_t)4 * std::max<long long>(net->n_params, 1) * sizeof(float);
            const hipError_t e = hipMalloc((void**)&net->mom, bytes);
            if (e != hipSuccess) {
                net->mom = nullptr;
                return fail(net, e == hipErrorOutOfMemory ? SNN_ENOMEM : SNN_EDEVICE, "hipMalloc: %s",
                            hipGetErrorString(e));
            }
            HIP_TRY(net, hipMemsetAsync(net->mom, 0, bytes, net->stream));
            net->adam_steps = 0;
        }
        const long long k = ++net->adam_steps;
        a.b1 = o->beta1;
        a.b2 = o->beta2;
        a.one_m_b1 = (float)(1.0 - (double)o->beta1);
        a.one_m_b2 = (float)(1.0 - (double)o->beta2);
        a.eps = o->eps;
        a.c1 = (float)(1.0 / (1.0 - pow((double)o->beta1, (double)k)));
        a.c2 = (float)(1.0 / (1.0 - pow((double)o->beta2, (double)k)));
        a.mom = net->mom;
    }
    HIP_TRY(net, launch_optimizer(a, net->stream));
    return SNN_OK;
}

extern "C" int snn_optimizer_reset(snn_net* net) {
    if (!net) return SNN_EINVAL;
    net->err[0] = 0;
    net->adam_steps = 0;
    if (net->mom)
        HIP_TRY(net, hipMemsetAsync(net->mom, 0,
                                    (size_t)4 * std::max<long long>(net->n_params, 1) * sizeof(float),
                                    net->stream));
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

extern "C" int snn_get_record_currents(const snn_net* net, int32_t layer, float* I) {
    if (!net || layer < 1 || layer >= net->t.L || net->t.kind[layer] != SNN_LIF || !I)
        return SNN_EINVAL;
    if (!net->fwd_ok) return SNN_ESTATE;
    snn_net* m = const_cast<snn_net*>(net);
    const Topo& t = net->t;
    const size_t n = (size_t)t.B * t.cap;
    if (n == 0) return SNN_OK;
    HIP_TRY(m, hipMemcpyAsync(I, net->rec_I + (size_t)t.lif[layer] * n, n * sizeof(float),
                              hipMemcpyDeviceToDevice, net->stream));
    HIP_TRY(m, hipStreamSynchronize(net->stream));
    return SNN_OK;
}

extern "C" int snn_get_stats(const snn_net* net, snn_stats* out) {
    if (!net || !out) return SNN_EINVAL;
    *out = net->stats;
    return SNN_OK;
}

extern "C" const char* snn_last_error(const snn_net* net) { return net ? net->err : g_create_err; }

extern "C" void snn_destroy(snn_net* net) {
    if (!net) return;
    (void)hipStreamSynchronize(net->stream);
    if (net->aux) (void)hipStreamSynchronize(net->aux);
    free_all(net);
    free(net);
}
