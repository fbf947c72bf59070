// Internal types shared by the host side and the kernels of libsnn (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "snn.h"

#define SNN_MAXP (2 * SNN_MAX_LAYERS)

// Device status word, one per handle.
struct DevStatus {
    int bad_input;                 // input spike list or labels failed validation
    int overflow;                  // some record count exceeded the capacity
    unsigned long long clamped;    // delays clamped while rounding
    unsigned long long degenerate; // skipped jumps (I- <= theta)
    unsigned long long layer_spikes[SNN_MAX_LAYERS];  // per LIF layer, all samples
};

// Topology and constants, passed by value to every kernel.
struct Topo {
    int L, P, B, T, S, cap, loss, n_in;
    int n_lif, lif_total;              // LIF layers, neurons over all LIF layers
    float alpha, beta, gamma, cc, theta, rscale, tau_s, dt;
    int n[SNN_MAX_LAYERS];
    int kind[SNN_MAX_LAYERS];
    int lif[SNN_MAX_LAYERS];           // index among LIF layers, -1 otherwise
    int lif_off[SNN_MAX_LAYERS];       // offset of a LIF layer among all LIF neurons
    int ring_lds[SNN_MAX_LAYERS];      // float offset of the layer's ring in LDS, -1: global
    int pre[SNN_MAXP], post[SNN_MAXP];
    long long woff[SNN_MAXP];          // offset of projection p in flat parameter arrays
};

struct FwdArgs {
    Topo t;
    const float* W[SNN_MAXP];
    const uint8_t* slot;               // flat [params]
    float* ring[SNN_MAX_LAYERS];       // global rings [B][S][n_l] (layers not in LDS)
    const int* in_neuron;
    const int* in_idx;                 // [B][T+1] first input event of each step
    int* out_count[SNN_MAX_LAYERS];    // caller's records, by layer index
    int* out_step[SNN_MAX_LAYERS];
    int* out_neuron[SNN_MAX_LAYERS];
    int* rec_n;                        // [n_lif][B][cap] internal neuron index
    float* rec_I;                      // [n_lif][B][cap] I- at the spike
    int* rec_idx;                      // [n_lif][B][T+1] first record of each step
    float* z;                          // [B][C]
    int* nstar;                        // [B][C]
    float* Vf;                         // [B][sum n_l] final state
    float* If;
    DevStatus* st;
    int mask_off;                      // byte offset of the ballot masks in LDS
};

struct BwdArgs {
    Topo t;
    const float* W[SNN_MAXP];
    const uint8_t* slot;
    float* ring[SNN_MAX_LAYERS];       // global adjoint rings [B][S][n_l] (layers not in LDS)
    const int* in_neuron;
    const int* in_idx;
    const int* rec_n;
    const float* rec_I;
    float* rec_D;                      // [n_lif][B][cap] lambda_V jump of each spike
    const int* rec_idx;
    const float* src;                  // [B][C] loss source per step (sum) or at n* (max)
    const int* nstar;
    double* SU;                        // [params] sum of lambda_I at arrivals
    double* SD;                        // [params] sum of w (lambda_I - lambda_V) at arrivals
    DevStatus* st;
    int acc_off;                       // byte offset of the fp64 jump sums in LDS
};

// Kernel launchers (snn_kernels.hip).
hipError_t launch_reset_status(DevStatus* st, hipStream_t s);
hipError_t launch_validate(const int* off, const int* step, const int* neuron, int nnz, int B, int T,
                           int n_in, const int* labels, int C, DevStatus* st, hipStream_t s);
hipError_t launch_step_index(const int* off, const int* step, int B, int T, int* idx,
                             const DevStatus* st, hipStream_t s);
hipError_t launch_round_delays(const float* const* D, const long long* woff, const long long* cnt,
                               int P, int max_delay, uint8_t* slot, DevStatus* st, hipStream_t s);
hipError_t launch_forward(const FwdArgs& a, int threads, size_t lds, hipStream_t s);
hipError_t launch_loss(const float* z, const int* labels, const int* nstar, int B, int C, int loss,
                       float rscale, float tau_m, float* loss_out, float* src, const DevStatus* st,
                       hipStream_t s);
hipError_t launch_fill_f64(double* p, long long n, hipStream_t s);
hipError_t launch_backward_a(const BwdArgs& a, int threads, size_t lds, hipStream_t s);
hipError_t launch_backward_b(const BwdArgs& a, int threads, size_t lds, hipStream_t s);
hipError_t launch_finalize(const double* SU, const double* SD, float* const* dW, float* const* dD,
                           const long long* woff, const long long* cnt, int P, float tau_s, float dt,
                           hipStream_t s);
hipError_t launch_copy_state(const float* src, int stride, int off, int n, int B, float* dst,
                             hipStream_t s);
hipError_t set_kernel_lds_limits(size_t bytes);
