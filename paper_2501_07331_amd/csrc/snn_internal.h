// Internal types shared by the host side and the kernels of libsnn (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "snn.h"

#define SNN_MAXP (2 * SNN_MAX_LAYERS)
#define SNN_MAX_LIF (SNN_MAX_LAYERS - 2)  // LIF layers are 1 .. L-2

// Per-step spike table of a LIF layer, one row per (sample, step):
// [spikes at the step, record index of its first spike, first SNN_STEP_IDS
// spiking neurons ascending, padding]; entries past the count are stale.
#define SNN_STEP_IDS 16
#define SNN_STEP_ROW 20

// Device status word, one per handle.
struct DevStatus {
    int bad_input;                   // input spike list or labels failed validation
    int overflow;                    // some record count exceeded the capacity
    unsigned long long clamped;      // delays clamped while rounding
    unsigned long long degenerate;   // skipped jumps (I- <= theta)
    unsigned long long layer_spikes[SNN_MAX_LAYERS];   // per LIF layer, all samples
    double reg_loss;                 // spike-count penalty of the last forward
    int cl_abort;                    // a cluster exchange gave up waiting (the results are void)
};

// Topology, constants and the LDS plan, passed by value to every kernel.
struct Topo {
    int L, P, B, T, S, cap, loss, n_in;   // S: the deepest delay ring (max_delay + 1)
    int n_lif, lif_total, maxn;        // LIF layers, LIF neurons, widest non-input layer
    int out_l;                         // the output layer (L - 1): LI readout, or LIF (spike-time loss)
    int out_lif;                       // 1: the output layer is LIF (SNN_LOSS_DMSE)
    int out_p;                         // the projection into the readout layer
    float alpha, beta, gamma, cc, theta, rscale, tau_s, dt;
    int n[SNN_MAX_LAYERS];
    int kind[SNN_MAX_LAYERS];
    int lif[SNN_MAX_LAYERS];           // index among LIF layers, -1 otherwise
    int lif_off[SNN_MAX_LAYERS];       // offset of a LIF layer among all LIF neurons
    int pre[SNN_MAXP], post[SNN_MAXP];
    long long woff[SNN_MAXP];          // offset of projection p in flat parameter arrays
    int dmax[SNN_MAXP];                // largest delay slot of projection p (its clamp)
    int Sp[SNN_MAXP];                  // delay-ring slots of projection p: dmax + 1
    int Sb[SNN_MAX_LAYERS];            // adjoint-ring slots of a LIF layer: the largest Sp of
                                       // the LIF-pre projections into it (0: no such ring)
    // forward delay ring of projection p (LIF pre and LIF post): LDS float
    // offset, or -1 for the global ring [B][S][n_post]
    int fring[SNN_MAXP];
    // backward ring of lambda_I - lambda_V (fp64) of a LIF layer read by
    // LIF-pre projections: LDS byte offset, or -1 for the global ring [B][Sb][n]
    int bring[SNN_MAX_LAYERS];
};

// Cluster mode of the per-sample cores, for layers whose rings do not fit in
// one workgroup's LDS: G workgroups of one wave serve one sample, workgroup g
// owning neurons [64 g, 64 g + 64) of every LIF layer and the LDS ring
// columns of its neurons.  One launch covers the samples [b0, b0 + gridDim.x
// / G).  Per step (forward) or per round of spikes (backward) the workgroups
// of a sample exchange data through device memory as 64-bit words, each a
// 32-bit payload with a 32-bit tag in the high half: agent-scope atomic
// stores and loads (coherent across the XCDs' L2 caches), so a word is
// either old or whole, and a reader knows it is current when its tag is.
// Tags are odd and advance by 2 per exchange (tag0 at the first), so the
// zeroed buffer never matches and no stale word of an earlier call does.
struct ClusterArgs {
    int G;                             // workgroups per sample; 0: one workgroup per sample
    int b0;                            // first sample of this launch
    unsigned tag0;                     // tag of the first exchange of this launch
    unsigned long long* x;             // exchange words, [clusters][2 (parity)][words per exchange]
};

// Input projection arrivals: A_in[b][n][j] = sum, in emission order, of the
// input-projection weights arriving at post j of layer 1 at step n.
struct InScanArgs {
    int B, T, S, n_in, n1, TB;         // S: ring slots of the input projection; TB: step span
                                       // of an 8-event chunk on the fast path; the LDS ring
                                       // holds S + TB - 1 arrival steps
    const uint2* ws0;                  // input projection (weight bits, slot) [n_in][n1]
    const int* in_neuron;
    const int* in_step;
    const int* in_idx;                 // [B][T+1] first input event of each step
    float* A_in;                       // [B][T][n_1]
    const DevStatus* st;
};

// Spikes per step of a LIF layer whose data the backward core prefetches a
// step ahead (more are loaded in further rounds), by LIF layer count; 16
// covers nearly every step of a 256-neuron layer at 14 spikes per neuron
// while its input is active (8 left a quarter of them to an extra round).
constexpr int bwd_prefetch(int n_lif) { return n_lif == 1 ? 16 : 4; }
// Spikes per layer and round of the backward core in cluster mode: a round
// costs one exchange between the workgroups of a sample.
constexpr int kClKC = 32;

// One LIF layer as seen by the forward core.
struct FwdLayer {
    int n;
    int nin;                           // projections into the layer, in projection order:
    int in_l[2];                       //   source LIF layer (0-based), -1: the input projection
    int in_pp[2];                      //   index among the source layer's LIF-post projections
    int in_S[2];                       //   LIF sources: that projection's ring slots,
    int in_ring_lds[2];                //   its ring (LDS float offset, or the HBM ring
    float* in_ring[2];                 //   [B][S+1][n])
    int npost;                         // LIF-post projections out of the layer (recurrent, then
                                       // feed-forward); entries past npost repeat a valid one
    int nq[2];                         //   post neurons
    int npre[2];                       //   rows of ws (the presynaptic layer's neurons)
    int S[2];                          //   ring slots (the projection's largest delay + 1)
    int ring_lds[2];                   //   delay ring [S+1][nq] (row S: dummy): LDS float offset,
    float* ring[2];                    //   or the HBM ring [B][S+1][nq]
    const uint2* ws[2];                //   (weight bits, slot) [n][nq]
    int* rec_n;                        // [B][cap] records: neuron, step, I-
    int* rec_s;
    float* rec_I;
    int* rec_idx;                      // [B][T+1] first record of each step
    int* rec_cnt;                      // [B]
    int* steptab;                      // [B][T][SNN_STEP_ROW]
    int* ncount;                       // [n] spikes per neuron over the batch (added), or NULL
    int* out_count;                    // caller's records: [B], [B][cap], [B][cap]
    int* out_step;
    int* out_neuron;
};

struct CoreFwdArgs {
    int B, T, cap, NW, n1, nstate;
    float alpha, beta, gamma, theta;
    FwdLayer ly[SNN_MAX_LIF];
    int soff[SNN_MAX_LIF];             // offset of each LIF layer in the [B][nstate] final state
    const float* A_in;                 // [B][T][n_1] input-projection arrivals
    float* Vf;                         // [B][nstate] final state
    float* If;
    DevStatus* st;
    int mask_off;                      // byte offset of the ballot masks [3][NL][NW] in LDS
    int ids_off;                       // byte offset of the step's spike lists [NL][64 NW] in LDS
    // the LI readout fused into the core as one extra wave (ro_C > 0): lane
    // k < ro_C owns output k; arrivals in an LDS ring [ro_S + 1][ro_C] (row
    // ro_S: dummy) at byte offset ro_off
    int ro_C, ro_feed, ro_nfeed, ro_S, ro_off, ro_loss;
    float ro_scale;
    const uint2* ro_ws;                // readout projection (weight bits, slot) [ro_nfeed][ro_C]
    float* z;                          // [B][C]
    int* nstar;                        // [B][C]
    ClusterArgs cl;                    // cluster mode (cl.G > 0): every ring in LDS, row width 64
};

struct ReadoutArgs {
    Topo t;
    const uint2* ws;                   // projection into the readout layer (weight bits, slot)
    const float* A_in;                 // arrivals when the readout is fed by the inputs
    const int* rec_n;                  // records of the layer feeding the readout
    const int* rec_s;
    const int* rec_idx;
    float* table;                      // global arrival table [B][T][C] if not in LDS
    float* z;                          // [B][C]
    int* nstar;                        // [B][C]
    float* Vf;
    float* If;
    int table_lds;                     // LDS float offset of the [T][C] table, -1: global
    const DevStatus* st;
};

// Readout adjoint: lambda of the LI layer from its loss source, trajectories,
// and the readout part of the jump sum of every spike of the feeding layer.
// The backward pass is fp64 throughout: constants from fp64 host arithmetic,
// adjoints, trajectories, rings, jump sums and gradient sums.
struct ReadoutBwdArgs {
    int B, T, C, cap, loss;
    double alpha, beta, cc;
    int LC, nch;                       // reverse-time chunks: nch chunks of LC steps
    double P11, P12, P22;              // M^LC, M = [[beta, cc], [0, alpha]] acting on (lambda_I, lambda_V)
    const uint2* ws;                   // [n_feed][C] (weight bits, slot)
    const int* rec_n;                  // records of the feeding LIF layer [B][cap], or NULL
    const int* rec_s;
    const int* rec_cnt;                // [B]
    const int* nstar;                  // [B][C]
    const double* src;                 // [B][C] loss source on lambda_V per step (sum) or at n*
    double2* traj;                     // [B][T][C] (lambda_I, lambda_I - lambda_V)
    double* A2;                        // [B][cap]
    int tab_lds;                       // 1: the [T][C] table of lambda_I - lambda_V lives in LDS
};

// One LIF layer as seen by the backward core.
struct BwdLayer {
    int n, lif_off;
    int S;                             // adjoint-ring slots
    int ring_lds;                      // LDS byte offset of the adjoint ring [S][n] (fp64); -1
                                       // global; -2 none
    double* ring;                      // global adjoint ring [B][S][n] when ring_lds == -1
    int npost;                         // LIF-post projections out of this layer: the recurrent
                                       // one, then the feed-forward one (projection order); the
                                       // entries past npost repeat a valid projection (loads stay
                                       // in bounds; their contributions are masked)
    int nq[2];                         // their post layer's neurons,
    int npre[2];                       //   rows of ws (an entry past npost may have fewer than n),
    int qS[2];                         //   adjoint-ring slots of the post layer,
    int qring_lds[2];                  //   its adjoint ring (LDS byte offset, or -1: global qring)
    double* qring[2];
    const uint2* ws[2];                //   (weight bits, slot) [n][nq]
    const float* recI;                 // [B][cap] I- of the records
    const int* recn;                   // [B][cap] neuron of the records
    const int* steptab;                // [B][T][SNN_STEP_ROW] per-step spike table
    const double* A2;                  // [B][cap] extra jump numerator per record (the readout
                                       // part of the jump sums, spike-time loss terms), or NULL
};

struct CoreBwdArgs {
    int B, T, cap, NW, lif_total;
    double alpha, beta, cc, theta;
    BwdLayer ly[SNN_MAX_LIF];
    double2* traj;                     // [B][T][lif_total] (lambda_I, lambda_I - lambda_V)
    DevStatus* st;
    int part_off;                      // LDS byte offset of the partial jump sums
    ClusterArgs cl;                    // cluster mode (cl.G > 0): adjoint rings in LDS, row width 64
    int cl_off;                        // cluster mode: LDS byte offset of the exchange staging (shares
                                       // [NL NP][kClKC][4] fp64, slot totals [NL kClKC] fp64, own
                                       // positions [NL][64] int, abort flag)
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
    unsigned short* g_step;            // steps (< 65536), grouped by neuron
    int stage_cap;                     // spikes of a sample staged in LDS (more: sorted in place)
    const DevStatus* st;
};

// The projections into one post layer, for the gradient pass.
struct GradGroup {
    int nq;                            // post neurons
    int jb;                            // blocks of J posts
    int units;                         // (4-block line group, sample block) units, rounded up to 8
    int out;                           // 1: the readout layer (trajectories tu_out / td_out)
    int off;                           // neuron offset of the layer in its trajectory array
    int np;                            // projections into the layer (1 or 2), in projection order
    int p[2];
    int npre[2];
    int pre[2];                        // their presynaptic layer
    int blk0;                          // first workgroup of the group
};

struct GradArgs {
    int B, T, SB, bs, lif_total, C, ngroups, nblk;
    int TW;                            // trajectory window: steps staged in LDS at a time
    int spcap;                         // LDS capacity for a sample's spike steps (16-bit), 0: none
    int glcap;                         // LDS ints for a sample's spike-list offsets (multiple of 4)
    float tau_s, dt;
    long long nparams;
    const double2* tr_lif;             // [B][T][lif_total] (lambda_I, lambda_I - lambda_V)
    const double2* tr_out;             // [B][T][C]
    const uint2* ws;                   // flat [params] (weight bits, slot)
    long long woff[SNN_MAXP];
    const int* g_off[SNN_MAX_LAYERS];  // per presynaptic layer: [B][n+1]
    const unsigned short* g_step[SNN_MAX_LAYERS];
    GradGroup grp[SNN_MAX_LAYERS];
    double* part;                      // [SB][2][nparams] per sample block (SB > 1)
    float* dW[SNN_MAXP];
    float* dD[SNN_MAXP];
};

// One optimiser step (snn_optimizer_step): rates per projection, constants
// rounded to fp32 on the host.
struct OptArgs {
    int P, kind;
    long long nparams;
    long long woff[SNN_MAXP];
    float* W[SNN_MAXP];
    float* D[SNN_MAXP];
    const float* dW[SNN_MAXP];
    const float* dD[SNN_MAXP];
    float lr_w[SNN_MAXP], lr_d[SNN_MAXP];
    float b1, b2, one_m_b1, one_m_b2, eps, c1, c2;
    float d_min, d_max;
    float* mom;                        // Adam: [4][nparams] (m_w, v_w, m_d, v_d)
};

// Kernel launchers (snn_forward.hip, snn_backward.hip, snn_optim.hip).
hipError_t launch_reset_status(DevStatus* st, hipStream_t s);
hipError_t launch_validate(const int* off, const int* step, const int* neuron, int nnz, int B, int T,
                           int n_in, const int* labels, int C, DevStatus* st, hipStream_t s);
hipError_t launch_step_index(const int* off, const int* step, int B, int T, int* idx,
                             const DevStatus* st, hipStream_t s);
hipError_t launch_round_delays(const float* const* D, const float* const* W, const long long* woff,
                               const long long* cnt, int P, const int* dmax, uint8_t* slot, uint2* ws,
                               DevStatus* st, hipStream_t s);
hipError_t launch_input_scan(const InScanArgs& a, size_t lds, hipStream_t s);
hipError_t launch_forward_core(const CoreFwdArgs& a, int n_lif, int threads, size_t lds,
                               hipStream_t s);
hipError_t launch_readout_forward(const ReadoutArgs& a, int threads, size_t lds, hipStream_t s);
hipError_t launch_loss(const float* z, const int* labels, int B, int C, int loss, float rscale,
                       float tau_m, float* loss_out, double* src, const DevStatus* st, hipStream_t s);
hipError_t launch_copy_state(const float* src, int stride, int off, int n, int B, float* dst,
                             hipStream_t s);
hipError_t launch_readout_adjoint(const ReadoutBwdArgs& a, int threads, size_t lds, hipStream_t s);
hipError_t launch_backward_core(const CoreBwdArgs& a, int n_lif, int threads, size_t lds,
                                hipStream_t s);
hipError_t launch_group(const GroupArgs& a, int B, hipStream_t s);
hipError_t launch_gradients(const GradArgs& a, int J, int KL, int threads, size_t lds, hipStream_t s);
hipError_t launch_grad_reduce(const GradArgs& a, int P, hipStream_t s);
hipError_t launch_optimizer(const OptArgs& a, hipStream_t s);
hipError_t launch_dmse_loss(const int* rec_cnt, const int* rec_s, const int* rec_n, int cap,
                            const int* labels, int B, int C, int T, float dt, float delta, float* z,
                            float* loss_out, double* xlp, const DevStatus* st, hipStream_t s);
hipError_t launch_add_lp(double* dst, const double* base, const float* dlp, const double* nterm,
                         const int* rec_n, const int* cnt, int B, int cap, hipStream_t s);
// Spike-count regulariser: per LIF layer l with rho[l] != 0 and neuron i,
// cbar = ncount[i] / B, nterm[i] = -rho (cbar - nu) / B, and the penalty
// sum (rho / 2) (cbar - nu)^2 into st->reg_loss.
struct RegArgs {
    int nl, B;
    int n[SNN_MAX_LIF];
    double rho[SNN_MAX_LIF];
    const int* ncount[SNN_MAX_LIF];
    double* nterm[SNN_MAX_LIF];
    double nu;
    DevStatus* st;
};
hipError_t launch_spike_reg(const RegArgs& a, hipStream_t s);
hipError_t launch_zero_ints(int* p, long long n, hipStream_t s);
hipError_t set_forward_lds_limits(size_t bytes, int* bad);
hipError_t set_core_lds_limits(size_t bytes, int* bad);
bool launch_forward_core_256(const CoreFwdArgs& a, int n_lif, int np, bool rl, int threads,
                             size_t lds, hipStream_t s);
bool launch_forward_core_1024(const CoreFwdArgs& a, int n_lif, int np, bool rl, int threads,
                              size_t lds, hipStream_t s);
hipError_t set_core_lds_limits_256(size_t bytes, int* bad);
hipError_t set_core_lds_limits_1024(size_t bytes, int* bad);
hipError_t set_backward_lds_limits(size_t bytes, int* bad);
// Cluster mode (CoreFwdArgs::cl, CoreBwdArgs::cl): grid = clusters x G
// workgroups of 64 (1 + LIF -> LIF projections) threads (a neuron wave and
// one wave per ring), launched cooperatively; occupancy in workgroups per CU.
hipError_t launch_forward_core_cluster(const CoreFwdArgs& a, int n_lif, int np, int grid, int threads,
                                       size_t lds, hipStream_t s);
hipError_t forward_cluster_occupancy(int n_lif, int np, int threads, size_t lds, int* blocks_per_cu);
hipError_t set_core_lds_limits_cl(size_t bytes, int* bad);
hipError_t launch_backward_core_cluster(const CoreBwdArgs& a, int n_lif, int np, int grid, int threads,
                                        size_t lds, hipStream_t s);
hipError_t backward_cluster_occupancy(int n_lif, int np, int threads, size_t lds, int* blocks_per_cu);
hipError_t launch_clear_abort(DevStatus* st, hipStream_t s);
