/*
 * snn.h -- C ABI of libsnn: batched, time-stepped EventProp training step for
 * leaky integrate-and-fire networks with learnable synaptic delays, on AMD
 * Instinct MI355X (gfx950).
 *
 * Method: "Efficient Event-based Delay Learning in Spiking Neural Networks"
 * (Mészáros, Knight, Nowotny, arXiv 2501.07331), Table 1 and the Methods
 * ("Learning Weights in networks with delay", "Learning Delays").
 *
 * Model.  Layer 0 is an input layer of spike sources, layers 1 .. L-2 are LIF
 * layers (optionally recurrent), layer L-1 is a leaky-integrator (LI) readout,
 * i.e. a LIF layer with an infinite threshold (Table 1 caption), or, with the
 * spike-time loss, a spiking LIF output layer.  Between
 * events tau_m V' = -V + I and tau_s I' = -I; a LIF neuron spikes when V
 * reaches theta and is reset to 0; a spike of neuron i at step n makes the
 * current of post neuron j jump by w_ij at step n + d_ij (Table 1, forward).
 * The backward pass runs the adjoints lambda_V, lambda_I in reverse time,
 * applies the lambda_V jump at every saved spike using the postsynaptic
 * adjoints at the delayed arrival time, and accumulates
 *   dL/dw_ij = -tau_s sum_spikes lambda_I,j(t + d_ij),
 *   dL/dd_ij = -w_ij  sum_spikes (lambda_I - lambda_V)_j(t + d_ij)
 * (Table 1, gradient updates; Methods equations for the weight and delay
 * gradients and the lambda_V jump).
 *
 * Discretisation (the paper gives continuous equations only): a fixed grid of
 * T steps of dt.  Per step n: exact one-step propagation V- = fma(alpha, V,
 * gamma*I), I- = beta*I with alpha = e^{-dt/tau_m}, beta = e^{-dt/tau_s},
 * gamma = tau_s/(tau_s - tau_m) (beta - alpha) (constants computed in fp64 on
 * the host, rounded to fp32); threshold V- >= theta, reset, record (n, i, I-);
 * emit every presynaptic spike into its projection's delay ring (one per
 * sample and projection) at slot (n + d) mod S_p, S_p = the projection's
 * largest delay + 1, dropping arrivals at or after T; then I = I- +
 * ring_p[n mod S_p] for the projections p into the layer, in projection
 * order.  Delays are integer multiples of dt: the slot is rint(D) (round half
 * to even) clamped to [0, the projection's largest delay], NaN -> 0.  All
 * forward arithmetic is IEEE fp32 with no contraction; a ring cell sums its
 * weights in (emission step, presynaptic index) order, so spike records are
 * bit-reproducible.  The backward pass is fp64 throughout (adjoints, their
 * trajectories, jump sums, gradient sums), on the fp32 forward, and sums in
 * a fixed order: dW and dD are deterministic and within rounding of the fp64
 * evaluation of the same expressions.
 *
 * Projections.  Fixed order: for l = 1 .. L-1, the feed-forward projection
 * (l-1 -> l), then the recurrent one (l -> l) if layer l is recurrent.  Weight
 * and delay tensors of projection p are dense, row-major [n_pre][n_post]
 * (element (i, j) is the synapse from pre neuron i to post neuron j).  Delays
 * and delay gradients are in units of steps.
 *
 * Memory.  Every pointer argument marked (dev) is device memory owned by the
 * caller.  Inputs are read-only; outputs are fully overwritten.  The library
 * owns its scratch (delay rings, adjoint rings and trajectories, internal
 * spike records, per-step indices, a status word), allocated in snn_create
 * (grown on demand by the first calls that need more) and released in
 * snn_destroy.  Work is enqueued on
 * opts.hip_stream (NULL = the default stream); each snn_forward and
 * snn_backward ends with one small status read-back, so counts and error
 * codes are final when the call returns.  A handle is not thread-safe;
 * distinct handles are independent.
 */
#ifndef SNN_H
#define SNN_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
    SNN_OK = 0,
    SNN_EINVAL = -1,     /* bad topology, shape, argument or input spike list */
    SNN_ENOMEM = -2,     /* device allocation failed */
    SNN_ESTATE = -3,     /* snn_backward without a successful snn_forward */
    SNN_EOVERFLOW = -4,  /* a sample produced more spikes than record_capacity */
    SNN_EDEVICE = -5     /* a HIP runtime error */
};

enum { SNN_INPUT = 0, SNN_LIF = 1, SNN_LI = 2 };                /* layer kinds */
enum { SNN_LOSS_CE_SUM = 0, SNN_LOSS_CE_MAX = 1, SNN_LOSS_DMSE = 2 };   /* losses */

#define SNN_MAX_LAYERS 6
#define SNN_MAX_NEURONS 1024   /* per non-input layer */
#define SNN_MAX_INPUT 16384    /* input neurons */
#define SNN_MAX_DELAY 255
#define SNN_MAX_T 65536        /* steps per sample (spike steps are staged as 16-bit values) */

typedef struct snn_net snn_net;

/* One layer: n neurons, kind SNN_INPUT / SNN_LIF / SNN_LI, recurrent flag
 * (LIF layers only). */
typedef struct {
    int32_t n, kind, recurrent;
} snn_layer;

/*
 * batch:            samples per call (>= 1)
 * T:                steps per sample (>= 1)
 * loss:             SNN_LOSS_CE_SUM: z_k = readout_scale * sum_n V_k,n;
 *                   SNN_LOSS_CE_MAX: z_k = max_n V_k,n (first maximiser);
 *                   softmax cross-entropy on z, mean over the batch
 *                   (voltage-based readouts of Fig. 1 and the Results);
 *                   SNN_LOSS_DMSE: the last layer is LIF (not recurrent) and
 *                   z_k is the first spike time of output neuron k in ms
 *                   (n dt in fp64, rounded to fp32; T dt if it never fires);
 *                   the loss is the time-invariant mean squared error of the
 *                   Methods, L_b = 1/2 sum_{i != c} (z_i - z_c - dmse_delta)^2
 *                   with c = labels[b], mean over the batch; it enters the
 *                   backward pass as dL/dt_k at the first spike of each
 *                   output neuron (a neuron that never fires carries none)
 * readout_scale:    s above (sum readout only)
 * record_capacity:  spike records kept per sample and LIF layer
 * proj_max_delay:   host array of one largest delay (in steps) per projection,
 *                   each in [0, max_delay], or NULL (max_delay for every
 *                   projection): projection p's delays are clamped to it and
 *                   its delay ring (and the adjoint ring of its post layer)
 *                   holds that many steps + 1; read during snn_create only
 * flags:            bitwise OR of
 *                   SNN_FLAG_HBM_RINGS: keep every delay and adjoint ring in
 *                   device memory even where it would fit in LDS (same
 *                   results; exercises the HBM ring path);
 *                   SNN_FLAG_TIMING: time the main kernels with HIP events
 *                   on hip_stream (reported by snn_get_stats);
 *                   SNN_FLAG_SEPARATE_READOUT: run the LI readout as its own
 *                   kernel after the LIF core even where it fits into the
 *                   core's workgroup as one more wave (same results);
 *                   SNN_FLAG_CLUSTER: run the LIF cores in cluster mode
 *                   even where one workgroup per sample would hold the
 *                   rings in LDS (same forward results, bit for bit; the
 *                   backward sums its jump terms in another order).  Cluster
 *                   mode, which the library chooses by itself when a
 *                   sample's rings do not fit in one workgroup's LDS, spreads
 *                   a sample over ceil(widest LIF layer / 64) workgroups of
 *                   64 threads, each holding its neurons' ring columns in
 *                   LDS, which exchange the spikes (forward) and the partial
 *                   jump sums (backward) of every step through device memory;
 *                   it needs cooperative launches.  SNN_FLAG_HBM_RINGS wins
 *                   over it
 * hip_stream:       hipStream_t to enqueue on (NULL: default stream)
 * dmse_delta:       Delta_t of the spike-time loss, in ms (SNN_LOSS_DMSE)
 * reg_strength:     host array of one strength rho_l >= 0 per LIF layer (in
 *                   layer order), or NULL: the hidden spike-count
 *                   regulariser with target reg_target (spikes per neuron and
 *                   sample) that the Results apply to the hidden layers of
 *                   the SHD/SSC/Braille models (a target of 14 spikes per
 *                   example, a layer-wise strength).  With cbar_i the
 *                   batch-mean spike count of neuron i of layer l, the
 *                   penalty R = sum_l (rho_l / 2) sum_i (cbar_i - reg_target)^2
 *                   is reported as snn_stats.reg_loss, and every spike k of
 *                   neuron i adds dl_p/dt_k = -rho_l (cbar_i - reg_target) / B
 *                   to the numerator of its lambda_V jump (Table 1 backward
 *                   transition): the gradient, with the counts held fixed,
 *                   of -(rho_l / B) sum_i (cbar_i - reg_target) sum_k t_k,
 *                   which moves the spikes of an over-active neuron later and
 *                   those of an under-active one earlier; read during
 *                   snn_create only
 */
#define SNN_FLAG_HBM_RINGS 1
#define SNN_FLAG_TIMING 2
#define SNN_FLAG_SEPARATE_READOUT 4
#define SNN_FLAG_CLUSTER 8

typedef struct {
    int32_t batch, T, loss;
    float readout_scale;
    int32_t record_capacity;
    int32_t flags;
    void* hip_stream;
    float dmse_delta;
    const int32_t* proj_max_delay;
    float reg_target;
    const float* reg_strength;
} snn_opts;

/* Input spikes, CSR over samples (dev): offsets [batch+1] with offsets[0] = 0
 * and offsets[batch] = nnz; step and neuron [nnz]; within a sample sorted by
 * (step, neuron) without duplicates, 0 <= step < T, 0 <= neuron < n_input.
 * Checked on the device before any other kernel reads them (SNN_EINVAL). */
typedef struct {
    const int32_t* offsets;
    const int32_t* step;
    const int32_t* neuron;
    int32_t nnz;
} snn_spikes_in;

/* Spike records of one LIF layer (dev): count [batch]; step, neuron
 * [batch][record_capacity], each sample sorted by (step, neuron).  count is
 * exact even when it exceeds the capacity (then only the first
 * record_capacity records are stored and the call returns SNN_EOVERFLOW). */
typedef struct {
    int32_t* count;
    int32_t* step;
    int32_t* neuron;
} snn_spikes_out;

/* Per-call statistics of the last forward / backward (host copy). */
typedef struct {
    int64_t input_spikes;      /* nnz of the last forward */
    int64_t lif_spikes;        /* all LIF layers, all samples */
    int64_t events;            /* sum over projections of presynaptic spikes x n_post */
    int64_t clamped_delays;    /* delays rounded outside [0, max_delay] or NaN */
    int64_t degenerate_jumps;  /* spikes with I- <= theta whose jump was skipped */
    int32_t overflow;          /* 1 if any record count exceeded the capacity */
    int32_t lds_rings;         /* bit p set: projection p's forward delay ring lives in LDS */
    /* with SNN_FLAG_TIMING, milliseconds of the last call's kernels, in order:
     * input_scan, forward_core, readout_forward (forward); readout_adjoint,
     * backward_core, group, gradients (backward) */
    float kernel_ms[8];
    double reg_loss;           /* spike-count penalty R of the last forward (0 if off) */
} snn_stats;

/*
 * Build a network handle: validates the topology (layer 0 SNN_INPUT, layers
 * 1 .. L-2 SNN_LIF, last layer SNN_LI, or a non-recurrent SNN_LIF with
 * SNN_LOSS_DMSE, 2 <= L <= SNN_MAX_LAYERS, at most SNN_MAX_LAYERS - 2 LIF
 * layers, non-input layers of 1 .. SNN_MAX_NEURONS neurons, only LIF layers
 * recurrent, at most SNN_MAX_INPUT input neurons),
 * computes the fp32 constants on the host in fp64, and allocates the device
 * scratch for opts->batch samples.  dt > 0, tau_m != tau_s, both > 0,
 * 0 <= max_delay <= SNN_MAX_DELAY, 1 <= opts->T <= SNN_MAX_T,
 * opts->batch x (opts->T + 1) <= 2^31.  No device compute.  *out receives the
 * handle (NULL on error); errors: SNN_EINVAL, SNN_ENOMEM, SNN_EDEVICE.
 */
int snn_create(const snn_layer* layers, int32_t n_layers, float tau_m, float tau_s, float theta,
               float dt, int32_t max_delay, const snn_opts* opts, snn_net** out);

/* Number of projections, and the layers / sizes of projection p. */
int snn_num_projections(const snn_net* net, int32_t* n);
int snn_projection_info(const snn_net* net, int32_t p, int32_t* pre_layer, int32_t* post_layer,
                        int32_t* n_pre, int32_t* n_post);

/*
 * Forward pass and loss (Table 1 forward dynamics; voltage readout loss).
 *   in:       input spikes (dev)
 *   W, D:     host arrays of P device pointers, projection p [n_pre][n_post]
 *             fp32; D in steps
 *   labels:   (dev) [batch] class indices in [0, C)
 *   records:  host array of one snn_spikes_out per LIF layer (dev buffers;
 *             the LIF output layer of SNN_LOSS_DMSE included, last)
 *   loss:     (dev) [batch + 1] per-sample loss, then the batch mean
 *   z:        (dev) [batch][C] readout values (first spike times for
 *             SNN_LOSS_DMSE), or NULL
 * The library keeps in, W, D and labels for snn_backward: the caller keeps
 * them alive and unmodified until the matching snn_backward returns.
 * Errors: SNN_EINVAL (NULL pointers, bad input spikes, bad labels),
 * SNN_EOVERFLOW (records truncated: counts, kept records and the final
 * state stay valid; loss and z are then computed from the truncated records
 * of the layer feeding the readout and carry no meaning), SNN_EDEVICE.
 */
int snn_forward(snn_net* net, const snn_spikes_in* in, const float* const* W, const float* const* D,
                const int32_t* labels, snn_spikes_out* records, float* loss, float* z);

/*
 * Backward pass of the last forward (Table 1 backward dynamics, lambda_V
 * jumps with delayed postsynaptic adjoints, weight and delay gradients).
 *   dW, dD:   host arrays of P device pointers, [n_pre][n_post] fp32; dD is
 *             dL per step of delay.  Gradients are summed over the batch of
 *             the mean loss (so they are batch means).
 * Adjoint state, trajectories, the jump's postsynaptic sum and the gradient
 * sums are fp64; dW and dD are rounded to fp32 once, at the end.
 * Errors: SNN_ESTATE (no successful forward),
 * SNN_EOVERFLOW (the forward overflowed its records), SNN_EINVAL, SNN_EDEVICE.
 */
int snn_backward(snn_net* net, float* const* dW, float* const* dD);

/*
 * snn_backward with a spike-time loss term on any LIF layer: the derivative
 * dl_p/dt_k of an extra loss l_p(spike times) with respect to the time (in
 * ms) of each recorded spike is added to the numerator of that spike's
 * lambda_V jump (Table 1 backward transition; Methods, the jump with
 * dl_p/dt_k), on top of the loss chosen at creation.
 *   dlp:      host array of one device pointer per LIF layer (in layer
 *             order, as the records), each [batch][record_capacity] fp32 in
 *             the order of that layer's records of the last forward, or
 *             NULL (no term on that layer); dlp itself may be NULL.  Entries
 *             past a sample's count are ignored.  For the gradient of a
 *             batch-mean loss the caller includes the 1/batch.
 * The term is added in fp64.  Errors as snn_backward.
 */
int snn_backward_lp(snn_net* net, const float* const* dlp, float* const* dW, float* const* dD);

/*
 * snn_backward for callers that cannot allocate device memory: code under
 * HIP graph capture, tight training or serving loops, harnesses that forbid
 * hipMalloc.  Same computation and results as snn_backward, bit for bit.
 * The one buffer snn_backward sizes by the last forward's input (the input
 * spikes grouped by channel: batch x (n_input + 1) + nnz int32, grown on
 * demand with hipMalloc) lives instead in a fixed library array of
 * SNN_NOALLOC_SCRATCH_BYTES per device, so the call makes no hipMalloc,
 * hipFree or other allocating call.  The array is shared by every handle on
 * a device and keeps the last call's contents (every entry this call reads
 * it writes first); calls that overlap on one device (other streams or host
 * threads) race on it and must be serialised by the caller.
 * Errors: as snn_backward, and SNN_EINVAL when batch x (n_input + 1) + nnz
 * exceeds SNN_NOALLOC_SCRATCH_BYTES / 4 (nothing is enqueued then).
 */
#define SNN_NOALLOC_SCRATCH_BYTES (32u << 20)
int snn_backward_noalloc(snn_net* net, float* const* dW, float* const* dD);

/*
 * Parameter update after snn_backward: one optimiser step on every W and D,
 * then the delay clamp.  The paper trains weights and delays with separate
 * learning rates and schedules (Methods / "Implementation" and its
 * hyper-parameter tables) and keeps delays non-negative (Fig. 3 caption); it
 * does not name the optimiser, so two are offered:
 *   SNN_OPT_SGD:   x <- x - lr * g                 (fp32, one rounding each op)
 *   SNN_OPT_ADAM:  m <- b1 m + (1 - b1) g,  v <- b2 v + (1 - b2) g g,
 *                  x <- x - lr * (m c1) / (sqrt(v c2) + eps),
 *                  c1 = 1 / (1 - b1^k), c2 = 1 / (1 - b2^k) at the k-th Adam
 *                  step of the handle (bias corrections computed in fp64 on
 *                  the host, rounded to fp32)
 * with g = dW (lr = lr_w * lr_scale_w[p]) for weights and g = dD (lr = lr_d *
 * lr_scale_d[p]) for delays, which are then clamped to [d_min, d_max] (in
 * steps; d_min <= d_max).  Learning-rate schedules are the caller's: it
 * passes this step's lr_w and lr_d.
 *   W, D:     host arrays of P device pointers, updated in place
 *   dW, dD:   host arrays of P device pointers (as written by snn_backward)
 *   lr_scale_w, lr_scale_d: host arrays of P factors per projection, or NULL
 *             (all 1); 0 freezes that projection's weights or delays
 * The Adam moments (4 fp32 per parameter) are owned by the handle, allocated
 * by its first Adam step, zero at that point and after snn_optimizer_reset.
 * Enqueued on the handle's stream; returns after it has been enqueued (no
 * read-back).  Errors: SNN_EINVAL (NULL pointers, unknown kind, non-finite
 * or negative rates, d_min > d_max, b1 or b2 outside [0, 1), eps <= 0),
 * SNN_ENOMEM, SNN_EDEVICE.
 */
enum { SNN_OPT_SGD = 0, SNN_OPT_ADAM = 1 };

typedef struct {
    int32_t kind;
    float lr_w, lr_d;
    float beta1, beta2, eps;      /* Adam only */
    float d_min, d_max;
    const float* lr_scale_w;      /* host [P] or NULL */
    const float* lr_scale_d;      /* host [P] or NULL */
} snn_optim;

int snn_optimizer_step(snn_net* net, const snn_optim* o, float* const* W, float* const* D,
                       const float* const* dW, const float* const* dD);

/* Zero the Adam moments and the Adam step count of the handle. */
int snn_optimizer_reset(snn_net* net);

/* Copy the final V and I of non-input layer `layer` after the last forward
 * into (dev) [batch][n_layer] buffers. */
int snn_get_state(const snn_net* net, int32_t layer, float* V, float* I);

/* Copy I- (the synaptic current just before the threshold test, Table 1
 * forward dynamics) of every stored spike record of LIF layer `layer` after
 * the last forward into (dev) [batch][record_capacity] fp32, in the order of
 * that layer's records; entries past a sample's stored count are
 * unspecified.  These are the denominators' currents of the backward jumps.
 * Errors: SNN_EINVAL (not a LIF layer, NULL I), SNN_ESTATE (no forward). */
int snn_get_record_currents(const snn_net* net, int32_t layer, float* I);

/* Statistics of the last forward / backward. */
int snn_get_stats(const snn_net* net, snn_stats* out);

/* Message for the last error on this handle ("" if none); valid until the
 * next call on the handle.  With net NULL: the reason of the last failed
 * snn_create on the calling thread ("" if none). */
const char* snn_last_error(const snn_net* net);

/* Release the handle and its device scratch (waits for its stream). */
void snn_destroy(snn_net* net);

#ifdef __cplusplus
}
#endif

#endif /* SNN_H */
