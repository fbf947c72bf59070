// Internal types shared by the host side and the kernels of libsnn (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "snn.h"

#define SNN_MAXP (2 * SNN_MAX_LAYERS)
#define SNN_MAX_INPUT 16384          // input neurons (per-sample spike grouping in LDS)

// Device status word, one per handle.
struct DevStatus {
    int bad_input;                   // input spike list or labels failed validation
    int overflow;                    // some record count exceeded the capacity
    unsigned long long clamped;      // delays clamped while rounding
    unsigned long long degenerate;   // skipped jumps (I- <= theta)
    unsigned long long layer_spikes[SNN_MAX_LAYERS];   // per LIF layer, all samples
};

// Topology, constants and the LDS plan, passed by value to every kernel.
struct Topo {
    int L, P, B, T, S, cap, loss, n_in;
    int n_lif, lif_total, maxn;        // LIF layers, LIF neurons, widest non-input layer
    int out_l;                         // the LI readout layer (L - 1)
    int out_p;                         // the projection into the readout layer
    float alpha, beta, gamma, cc, theta, rscale, tau_s, dt;
    int n[SNN_MAX_LAYERS];
    int kind[SNN_MAX_LAYERS];
    int lif[SNN_MAX_LAYERS];           // index among LIF layers, -1 otherwise
    int lif_off[SNN_MAX_LAYERS];       // offset of a LIF layer among all LIF neurons
    int pre[SNN_MAXP], post[SNN_MAXP];
    long long woff[SNN_MAXP];          // offset of projection p in flat parameter arrays
    // forward delay ring of projection p (LIF pre and LIF post): LDS float
    // offset, or -1 for the global ring [B][S][n_post]
    int fring[SNN_MAXP];
    // backward ring of lambda_I - lambda_V of a LIF layer read by LIF-pre
    // projections: LDS float offset, or -1 for the global ring [B][S][n]
    int bring[SNN_MAX_LAYERS];
};

// Input projection arrivals: A_in[b][n][j] = sum, in emission order, of the
// input-projection weights arriving at post j of layer 1 at step n.
struct InScanArgs {
    Topo t;
    const float* W0;
    const uint8_t* slot0;
    const int* in_neuron;
    const int* in_idx;                 // [B][T+1] first input event of each step
    float* A_in;                       // [B][T][n_1]
    const DevStatus* st;
    int nb;                            // posts per workgroup (ring [S][nb] in LDS)
};

struct CoreFwdArgs {
    Topo t;
    const float* W[SNN_MAXP];
    const uint8_t* slot;               // flat [params]
    float* ring[SNN_MAXP];             // global rings of LIF->LIF projections not in LDS
    const float* A_in;
    int* out_count[SNN_MAX_LAYERS];    // caller's records, by layer index
    int* out_step[SNN_MAX_LAYERS];
    int* out_neuron[SNN_MAX_LAYERS];
    int* rec_n;                        // [n_lif][B][cap] neuron
    int* rec_s;                        // [n_lif][B][cap] step
    float* rec_I;                      // [n_lif][B][cap] I- at the spike
    int* rec_idx;                      // [n_lif][B][T+1] first record of each step
    int* rec_cnt;                      // [n_lif][B] spikes per sample
    float* Vf;                         // [B][sum n_l] final state
    float* If;
    DevStatus* st;
    int mask_off;                      // byte offset of the ballot masks in LDS
};

struct ReadoutArgs {
    Topo t;
    const float* W;                    // projection into the readout layer
    const uint8_t* slot;
    const float* A_in;                 // arrivals when the readout is fed by the inputs
    const int* rec_n;                  // records of the layer feeding the readout
    const int* rec_s;
    const int* rec_idx;
    float* table;                      // global arrival table [B][T][C] if not in LDS
    float* z;                          // [B][C]
    int* nstar;                        // [B][C]
    float* Vf;
    float* If;
    // backward
    const float* src;                  // [B][C]
    float* tu;                         // [B][C][T] lambda_I of the readout
    float* td;                         // [B][C][T] lambda_I - lambda_V of the readout
    int table_lds;                     // LDS float offset of the [T][C] table, -1: global
    int red_off;                       // byte offset of the fp64 reduction scratch in LDS
    double* A2;                        // [B][cap] readout part of each feeding spike's jump sum
    const DevStatus* st;
};

struct CoreBwdArgs {
    Topo t;
    const float* W[SNN_MAXP];
    const uint8_t* slot;
    float* ring[SNN_MAX_LAYERS];       // global adjoint rings [B][S][n_l] (layers not in LDS)
    const int* rec_n;
    const float* rec_I;
    const int* rec_idx;
    const double* A2;                  // readout part of the jump sums of the last LIF layer
    float* tu;                         // [B][lif_total][T] lambda_I
    float* td;                         // [B][lif_total][T] lambda_I - lambda_V
    DevStatus* st;
    int acc_off;                       // byte offset of the fp64 jump sums in LDS
};

// Spikes of each sample grouped by presynaptic neuron, in step order.
struct GroupArgs {
    const int* off;                    // spikes of sample b start at off[b] (absolute index)
    const int* end;                    // [B+1] off (CSR) if cnt is NULL
    const int* cnt;                    // or [B] counts: spikes of b are [off[b], off[b] + cnt[b])
    int off_stride;                    // with cnt: off[b] = b * off_stride
    const int* step;                   // per spike
    const int* neuron;
    int n;                             // presynaptic neurons
    int* g_off;                        // [B][n+1] start of neuron i's steps (absolute index)
    int* g_step;                       // steps, grouped by neuron
    const DevStatus* st;
};

struct GradArgs {
    Topo t;
    const float* W[SNN_MAXP];
    const uint8_t* slot;
    const float* tu_lif;               // [B][lif_total][T]
    const float* td_lif;
    const float* tu_out;               // [B][C][T]
    const float* td_out;
    const int* g_off[SNN_MAX_LAYERS];  // per presynaptic layer: [B][n+1]
    const int* g_step[SNN_MAX_LAYERS];
    float* dW[SNN_MAXP];
    float* dD[SNN_MAXP];
    int blk[SNN_MAXP + 1];             // workgroups of projection p: [blk[p], blk[p+1]) = posts
};

// Kernel launchers (snn_kernels.hip).
hipError_t launch_reset_status(DevStatus* st, hipStream_t s);
hipError_t launch_validate(const int* off, const int* step, const int* neuron, int nnz, int B, int T,
                           int n_in, const int* labels, int C, DevStatus* st, hipStream_t s);
hipError_t launch_step_index(const int* off, const int* step, int B, int T, int* idx,
                             const DevStatus* st, hipStream_t s);
hipError_t launch_round_delays(const float* const* D, const long long* woff, const long long* cnt,
                               int P, int max_delay, uint8_t* slot, DevStatus* st, hipStream_t s);
hipError_t launch_input_scan(const InScanArgs& a, size_t lds, hipStream_t s);
hipError_t launch_forward_core(const CoreFwdArgs& a, int threads, size_t lds, hipStream_t s);
hipError_t launch_readout_forward(const ReadoutArgs& a, int threads, size_t lds, hipStream_t s);
hipError_t launch_loss(const float* z, const int* labels, int B, int C, int loss, float rscale,
                       float tau_m, float* loss_out, float* src, const DevStatus* st, hipStream_t s);
hipError_t launch_readout_adjoint(const ReadoutArgs& a, int threads, size_t lds, hipStream_t s);
hipError_t launch_backward_core(const CoreBwdArgs& a, int threads, size_t lds, hipStream_t s);
hipError_t launch_group(const GroupArgs& a, int B, hipStream_t s);
hipError_t launch_gradients(const GradArgs& a, int blocks, size_t lds, hipStream_t s);
hipError_t launch_copy_state(const float* src, int stride, int off, int n, int B, float* dst,
                             hipStream_t s);
hipError_t set_kernel_lds_limits(size_t bytes);
