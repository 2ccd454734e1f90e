/*
 * eprop.h -- C ABI of the MI355X (gfx950) online e-prop library.
 *
 * The library runs the per-timestep hot path of gradient-based synaptic
 * plasticity (arxiv 2501.11407) for recurrent spiking networks of LIF and
 * ALIF neurons: the synaptic drive, the neuron step with its surrogate
 * pseudo-derivative, the per-synapse eligibility-vector update and the
 * learning-signal-weighted gradient accumulation.
 *
 * The calls follow the paper's statement of the problem (Sec. III-A):
 *   - Eq. (1): a state recursion h_{t+1} = f(h_t, x_t, theta) driven by the
 *     inputs x_t  -> eprop_step / eprop_run_sequence;
 *   - Eq. (2): a loss that is a sum of per-step losses (softmax cross-entropy
 *     of a leaky non-spiking readout at every step);
 *   - Eq. (3) with the recursion of Eq. (5): the gradient accumulated forward
 *     in time, G_t = H_t G_{t-1} + F_t, with H_t restricted to its diagonal
 *     neuron-on-itself part (Sec. III-B), so that the state the library keeps
 *     does not depend on the sequence length  -> eprop_get_grads.
 *
 * Model (per layer, per batch element b, per step t; j = neuron, i = input):
 *   p^t      = [in^t ; z^{t-1}]            (in = x for layer 0, layer-1 spikes of
 *                                           the same step for layer 1; no z part
 *                                           when recurrent == 0)
 *   v^t_j    = alpha v^{t-1}_j + sum_i W_ji p^t_i - thr z^{t-1}_j
 *   a^t_j    = rho a^{t-1}_j + z^{t-1}_j ;  A_j = thr + beta_j a^t_j
 *              (beta_j = beta for j < n_adaptive, else 0)
 *   z^t_j    = [v^t_j - A_j > 0] ;  psi_j = (gamma/thr) max(0, 1 - |v_j - A_j|/thr)
 *   y^t      = kappa y^{t-1} + W_out z^t ;  loss += CE(softmax(y^t), label_b)
 * Gradient stops: the recurrent spikes z^{t-1} in the drive and the reset,
 * and (two layers) the layer-1 spikes fed to layer 2.  Each layer learns from
 * its own readout.  The gradient is dE/dW for E = sum_b sum_t sum_layers CE,
 * not averaged; the recurrent diagonal (self-connections) is reported as 0.
 *
 * Memory: every device buffer belongs to the caller.  The library works in
 * one caller-provided device workspace whose size depends on the shape but
 * not on the sequence length, and borrows the weight buffers until
 * eprop_destroy.
 *
 * Streams: every call that takes a context enqueues work on the stream given
 * to eprop_init and returns without waiting, except eprop_status and
 * eprop_profile_end, which wait for that stream.  A context belongs to one
 * stream and one host thread at a time.  Internally the forward and
 * coefficient kernels run on two streams of the context's own, joined to the
 * caller's stream by events: work enqueued on the caller's stream before a
 * call happens before it, and work enqueued after a call sees its results.
 */
#ifndef EPROP_H
#define EPROP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
#define EPROP_OK 0
#define EPROP_EINVAL (-1)   /* null pointer, bad dimension or constant, T < 1 */
#define EPROP_ENOSPACE (-2) /* workspace smaller than eprop_workspace_bytes */
#define EPROP_EDEVICE (-3)  /* HIP runtime or launch error; see eprop_last_error */
#define EPROP_ESTATE (-4)   /* context not initialised, or a device-side input error */

typedef struct eprop_ctx eprop_ctx; /* opaque, host-side */

/* Network shape and constants.  All constants are used as given, in fp32. */
typedef struct {
  int32_t n_layers;   /* 1, or 2 for a stack fed layer-1 spikes of the same step */
  int32_t batch;      /* 1 <= B <= 65535 */
  int32_t n_in;       /* inputs of layer 0, 1 .. 65536 */
  int32_t n_rec;      /* neurons per layer, 1 .. 8192 */
  int32_t n_out;      /* readout classes K, 1 .. 1024 */
  int32_t recurrent;  /* 1: presynaptic vector [in ; z^{t-1}], 0: in only */
  int32_t n_adaptive; /* neurons j < n_adaptive are ALIF (0 <= n_adaptive <= n_rec) */
  float alpha;        /* membrane decay exp(-dt/tau_m), Eq. (8a) */
  float rho;          /* adaptation decay */
  float kappa;        /* readout decay */
  float thr;          /* threshold theta > 0, also the reset amount */
  float beta;         /* threshold adaptation strength of ALIF neurons */
  float gamma;        /* surrogate height */
  int32_t reset_grad; /* 0: the reset path (own spike -> own membrane) is
                         gradient-stopped like the recurrent spikes; 1: it is
                         kept (Eq. 5 with the reset's terms in the membrane
                         row of H_I, Sec. III-C), so the membrane eligibility
                         is a third per-synapse trace; other values: -1 */
  int32_t neuron_model; /* 0: LIF/ALIF as above.  1: a two-compartment
                         neuron (n_adaptive must be 0; rho and beta unused):
                           d^t = alpha_d d^{t-1} + sum_i W_ji p^t_i + bap z^{t-1}
                           s^t = alpha s^{t-1} + coupling d^{t-1} - thr z^{t-1}
                           z^t = [s^t - thr > 0], psi from s^t - thr as above;
                         the own spike's path into the dendrite is kept in
                         the gradient (the soma reset follows reset_grad), so
                         H_I is a full 2x2 block per neuron (footnote of
                         Sec. III-C) and both eligibility components are
                         per-synapse traces */
  float alpha_d;      /* neuron_model 1: dendritic decay */
  float coupling;     /* neuron_model 1: dendrite -> soma coupling */
  float bap;          /* neuron_model 1: own spike -> dendrite */
} eprop_config;

/*
 * The neuron model's step, h^t = A h^{t-1} + b I^t + r z^{t-1} with the spike
 * argument u = c . h - thr, differentiated on the host by forward-mode dual
 * numbers (the automatic derivation of H_I and F_t of Sec. III-C for models
 * whose step is linear in the state): out[0..9] = A00 A01 A10 A11 b0 b1 r0 r1
 * c0 c1 for neurons j < n_adaptive (cls = 1) or the others (cls = 0), with
 * r the own-spike terms that stay in the gradient (the reset of component 0
 * only when reset_grad = 1), so that H_I^t = A + psi^{t-1} r c^T and
 * F_t = b p^t.  Host only.  Returns 0, or EPROP_EINVAL (invalid config, a
 * step that is not linear in its state).
 */
int eprop_neuron_coefficients(const eprop_config* cfg, int32_t cls, float* out);

/*
 * Bytes of device workspace a context with this shape needs; 0 if the
 * configuration is invalid.  There is no sequence-length argument: the
 * e-prop state is O(B * N_pre * N_post) and independent of T (Table I).
 */
size_t eprop_workspace_bytes(const eprop_config* cfg);

/*
 * Creates a context in the caller's device workspace (>= 256-byte aligned,
 * at least eprop_workspace_bytes(cfg) bytes) and copies the weights into it.
 *   d_weights: host array of 2*n_layers device pointers, per layer l:
 *     d_weights[2l]   = W     fp32 [n_rec][n_pre_l] row-major, n_pre_l =
 *                       n_in_l + (recurrent ? n_rec : 0), columns [W_in | W_rec]
 *     d_weights[2l+1] = W_out fp32 [n_out][n_rec] row-major
 *   The weights are read here and again by every eprop_reset, and must not be
 *   freed before eprop_destroy.
 *   hip_stream: a hipStream_t (NULL = the null stream).
 * State, traces and accumulators start at zero (the recursion of Eq. (5)
 * starts from G_0 = 0, Sec. III-A).  On success *out is the new
 * context and 0 is returned; on failure *out is NULL and the reason is in
 * eprop_last_error(NULL).
 */
int eprop_init(const eprop_config* cfg, void* d_workspace, size_t ws_bytes,
               const float* const* d_weights, void* hip_stream, eprop_ctx** out);

/*
 * One online e-prop step (one timestep) for every layer:
 *   d_x_t:     device uint8 [B][n_in]; a nonzero byte is an input spike
 *   d_labels:  device int32 [B], class of each batch element, in [0, n_out)
 *              (an out-of-range label is a device-side error reported by
 *              eprop_status; its step gets no target term)
 *   d_spikes_t: NULL, or device uint32 [n_layers][B][ceil(n_rec/32)] receiving
 *              the step's spikes, bit j%32 of word j/32
 * Updates the neuron state, the eligibility vectors and the gradient
 * accumulators in the workspace.
 */
int eprop_step(eprop_ctx* ctx, const uint8_t* d_x_t, const int32_t* d_labels,
               uint32_t* d_spikes_t);

/*
 * T >= 1 consecutive steps, equivalent to T calls of eprop_step:
 *   d_x: device uint8 [T][B][n_in];  d_labels: as for eprop_step, used at
 *   every step;  d_spikes: NULL or device uint32 [T][n_layers][B][ceil(n_rec/32)].
 * The steps are processed in blocks of consecutive timesteps: the forward
 * dynamics never read the eligibility vectors, so the network is run ahead
 * through a block and the traces then advance through all of its steps with
 * one pass over them.  Spike trains, neuron state and traces are identical
 * however a sequence is split into calls; the accumulated gradients agree up
 * to the order of floating-point summation (relative differences ~1e-7).
 * Identical call sequences give bit-identical results.
 */
int eprop_run_sequence(eprop_ctx* ctx, const uint8_t* d_x, int32_t T, const int32_t* d_labels,
                       uint32_t* d_spikes);

/*
 * How eprop_run_sequence splits a call into blocks (eprop_set_block_split).
 * The steps up to the next weight change (or the end of the call) form one
 * block when they number at most 256, else blocks of equal length (within a
 * step), at least two and each at most 512 steps, the block limit.  With
 * EPROP_SPLIT_AUTO (the default) a rough cost model of the shape may change
 * that in two places: a run of 128 to 256 steps is cut in two halves when the
 * forward steps of a half cost more than one more trace round trip; and a run
 * of more than 512 steps may start with a short block followed by blocks of
 * twice its length, one block more than the equal split, when starting the
 * first eligibility pass earlier saves more than the added round trip costs.
 * EPROP_SPLIT_EQUAL always takes the equal split.
 */
#define EPROP_SPLIT_AUTO 0
#define EPROP_SPLIT_EQUAL 1

/*
 * Sets the split mode of the context's later eprop_run_sequence calls (kept
 * over resets).  The split changes only the order of floating-point
 * summation in the gradients.  Returns 0, EPROP_EINVAL (unknown mode),
 * EPROP_ESTATE.
 */
int eprop_set_block_split(eprop_ctx* ctx, int32_t mode);

/*
 * The block lengths eprop_run_sequence uses for a call of T steps that starts
 * t0 steps after the last reset, with online application every `online_every`
 * steps (0: none), for the shape `cfg` and split `mode`.  Host only: touches
 * no device and no context.  Writes min(count, max_blocks) lengths to
 * `lengths` (host int32; may be NULL when max_blocks is 0) and returns the
 * count of blocks, or EPROP_EINVAL (invalid config or mode, T < 1, t0 < 0,
 * online_every < 0, max_blocks < 0, or lengths NULL with max_blocks > 0).
 */
int eprop_block_lengths(const eprop_config* cfg, int32_t T, int64_t t0, int32_t online_every,
                        int32_t mode, int32_t* lengths, int32_t max_blocks);

/*
 * Writes the gradient accumulated since the last reset, summed over batch
 * elements and steps:
 *   d_grads: host array of 2*n_layers device pointers, per layer l:
 *     d_grads[2l] = dE/dW fp32 [n_rec][n_pre_l] (layout of W; the recurrent
 *                   diagonal is 0), d_grads[2l+1] = dE/dW_out fp32 [n_out][n_rec]
 *   d_loss: NULL or device double[1] receiving E = sum of the per-step losses.
 * Accumulation happens in fp64 and is rounded to fp32 here.  The context
 * keeps accumulating; the caller synchronises the stream before reading.
 */
int eprop_get_grads(eprop_ctx* ctx, float* const* d_grads, double* d_loss);

/*
 * Starts a new sequence: zeroes neuron state, filters, eligibility vectors,
 * gradient and loss accumulators (G_0 = 0 and h_0 = 0 at the start of the
 * recursion of Eq. (1) and (5), Sec. III-A), and re-reads the weights and
 * any feedback matrices.
 */
int eprop_reset(eprop_ctx* ctx);

/*
 * Waits for the context's stream and reports device-side input errors seen
 * since the last reset: EPROP_ESTATE if a label was out of range, else 0 (or
 * EPROP_EDEVICE on a runtime error).
 */
int eprop_status(eprop_ctx* ctx);

/*
 * Learning signal through fixed feedback matrices instead of the readout
 * weights: L = B^T (softmax(y) - onehot(label)) per layer, the random-feedback
 * alternative to the readout's gradient that the source of the paper's
 * Sec. III-B names and sets aside.  Only the learning signal changes; the
 * readout, the loss and the readout gradient still use W_out.
 *   d_feedback: NULL (every layer back to B = W_out), or a host array of
 *     n_layers device pointers, each NULL (that layer: B = W_out) or B fp32
 *     [n_out][n_rec] row-major, the layout of W_out.
 * The matrices are read here (queued on the context's stream) and again by
 * every eprop_reset, must not be freed while set, and apply from the next
 * step on.  Nothing else is read or rewritten: the weights in use (with
 * online application, the updated ones) stay as they are.  With online
 * application the matrices keep their values while W and W_out change.
 * Returns 0, EPROP_ESTATE on an unusable context.
 */
int eprop_set_feedback(eprop_ctx* ctx, const float* const* d_feedback);

/*
 * Online weight application: the gradient is available at every step
 * (Sec. III-A), so the weights may change during the sequence.  Before the
 * step that follows every `every` steps counted from the last reset, the drive
 * and readout weights in use become W0 - lr * G rounded to the nearest
 * multiple of 2^-14 (ties to even; the grid keeps the drive's sums exact),
 * where W0 are the weights read at init or reset and G the gradient
 * accumulated since that reset (what eprop_get_grads would return); the
 * recurrent diagonal keeps W0.  The learning signal then uses the readout
 * weights in use at its step.  No update follows the last step run, and the
 * caller's weight buffers are not written (eprop_get_weights reads the ones in
 * use).  Feedback matrices set by eprop_set_feedback are not weights: they
 * keep their values.  every = 0 (the default) or lr = 0 turns it off; it applies from the
 * next step on and is kept over resets.  The blocks of eprop_run_sequence
 * end at the update steps, and the forward of the block after an update waits
 * for it.  Returns 0, EPROP_EINVAL (every < 0 or lr not finite), EPROP_ESTATE.
 */
int eprop_set_online(eprop_ctx* ctx, float lr, int32_t every);

/*
 * The weights in use (after any online updates), queued on the context's
 * stream: d_weights as eprop_init's (device pointers, layouts of W and W_out),
 * written, not read.  Returns 0, EPROP_EINVAL on a NULL pointer, EPROP_ESTATE.
 */
int eprop_get_weights(eprop_ctx* ctx, float* const* d_weights);

/* Frees the host-side context; the workspace and weights stay the caller's. */
void eprop_destroy(eprop_ctx* ctx);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid it): one whole sequence
 * without a caller workspace, creating no streams or events.  Equivalent to
 * eprop_init + eprop_run_sequence(d_x, T, d_labels, d_spikes) +
 * eprop_get_grads(d_grads, d_loss) + eprop_destroy, with the same kernels and
 * results, all queued on hip_stream (one stream: the forward of a block does
 * not overlap the eligibility pass of the one before).  Arguments as for
 * those calls; the weights are read on the stream.
 * The workspace is the library's static scratch, EPROP_STATIC_SCRATCH_BYTES
 * of device memory that every GPU the library runs on holds from the first
 * use of the library until the process ends.  On one stream nothing
 * overlaps, so a sequence here takes one set of per-block buffers, where
 * eprop_workspace_bytes counts the three a context pipelines with; shapes
 * whose workspace with one set exceeds the scratch return EPROP_ENOSPACE
 * (before any device call).  The device is the one current on the calling thread, which must be
 * the stream's.  Every call on one GPU uses that GPU's one scratch array:
 * calls that overlap on a GPU (queued on different streams without ordering,
 * or from several host threads) race; calls queued on one stream do not.
 * Each call clears what it needs itself.  Errors: eprop_last_error(NULL).
 */
#define EPROP_STATIC_SCRATCH_BYTES (256u << 20)
int eprop_sequence_static(const eprop_config* cfg, const float* const* d_weights,
                          const uint8_t* d_x, int32_t T, const int32_t* d_labels,
                          uint32_t* d_spikes, float* const* d_grads, double* d_loss,
                          void* hip_stream);

/*
 * Message of the last failure on ctx, or of the last failed eprop_init /
 * workspace query of this thread when ctx is NULL.  Never NULL.
 */
const char* eprop_last_error(const eprop_ctx* ctx);

/*
 * Kernel timing.  eprop_profile_begin makes the next calls record a pair of
 * HIP events, on the context's stream, around each launch of the eligibility
 * kernel (at most max_launches pairs; one launch advances the traces through
 * a block of consecutive timesteps).  eprop_profile_end waits for the stream
 * and returns the summed duration in milliseconds, the number of timed
 * launches and the number of timesteps they covered, then stops recording.
 */
int eprop_profile_begin(eprop_ctx* ctx, int32_t max_launches);
int eprop_profile_end(eprop_ctx* ctx, double* total_ms, int32_t* n_launches, int64_t* n_steps);

/*
 * Diagnostics: device address and shape of one internal per-neuron buffer of
 * layer `layer` as left by the last step, for checking intermediate values.
 *   which: 0 = v, 1 = a, 2 = psi, 3 = L (learning signal), 4 = y (readout)
 *   fp32, rows = B, row stride *ld elements, *cols valid columns.
 *   which = 5: two int32 (rows = 1, cols = ld = 2, any layer): [0] is 1 when
 *   every drive weight is k 2^-14 with integer |k| <= 32767, [1] the largest
 *   |k|.  Then every step with at most 2^24 / [1] active presynaptic inputs
 *   sums the weights as integers (each partial sum is then exact in fp32:
 *   the same result as the fp32 sum); other steps, and all steps when [0] is
 *   0, sum fp32 weights in ascending input order.  Valid once the work queued
 *   by init, reset or an online update has run.
 */
int eprop_debug_buffer(eprop_ctx* ctx, int32_t layer, int32_t which, const float** d_ptr,
                       int64_t* cols, int64_t* ld);

#ifdef __cplusplus
}
#endif

#endif /* EPROP_H */
