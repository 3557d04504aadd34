/*
 * hetpipe.h -- C ABI of the MI355X (gfx950) implementation of HetPipe's
 * data-parallel hot path: one pipeline stage's CNN training step and the
 * Wave Synchronous Parallel (WSP) weight update (HetPipe, arXiv 2005.14038).
 *
 * Objects
 *   hp_stage  one pipeline stage: a list of layers executed on one GPU
 *             (Sec. 3, pipelined model parallelism inside a virtual worker).
 *   hp_ps     the parameter server holding the global weights w_g and the
 *             global clock c_g (Sec. 5), resident in device memory.
 *   hp_vw     one virtual worker's WSP state for the stage: the ring of the
 *             s_local+1 live weight versions, the wave accumulator u~, the
 *             local clock and the pulled global clock (Sec. 4 and Sec. 5).
 *
 * Conventions for every call
 *   * All tensors are device pointers (HIP global memory) owned by the caller
 *     unless stated otherwise, and must stay valid until the work enqueued on
 *     the object's stream has completed.  Activations are NHWC fp32;
 *     parameters, gradients, ring versions, u~ and w_g are flat fp32 vectors
 *     in the stage's parameter layout (hp_stage_param_layout).
 *   * Every object is bound to the HIP stream given at creation; device work
 *     is enqueued asynchronously on it.  Clocks and protocol state live on the
 *     host and are updated synchronously by the calls.  No call synchronises
 *     the device except *_destroy.  Objects are not thread-safe.
 *   * Every call returns a status: HP_OK, HP_WOULD_BLOCK (hp_wsp_pull only) or
 *     a negative error.  Errors never abort; hp_last_error() describes the
 *     last error of the calling thread.
 */
#ifndef HETPIPE_H
#define HETPIPE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---------------------------------------------------------------- status */
#define HP_OK            0
#define HP_WOULD_BLOCK   1   /* pull gate closed: the clock bound needs other VWs' pushes */
#define HP_ERR_ARG     (-1)  /* NULL pointer, bad shape, bad layer description */
#define HP_ERR_STATE   (-2)  /* call out of protocol order (see each call) */
#define HP_ERR_HIP     (-3)  /* a HIP launch or runtime call failed */
#define HP_ERR_NOMEM   (-4)  /* device allocation failed */

/* ----------------------------------------------------------- layer kinds */
#define HP_CONV        1   /* C -> K channels, R x S window, stride, pad, optional bias */
#define HP_FC          2   /* C = in features (input flattened in (h,w,c) order), K = out */
#define HP_RELU        3
#define HP_MAXPOOL     4   /* R x S window, stride, pad; padded taps never win */
#define HP_BN          5   /* training-mode batch-norm over (n,h,w), C channels, eps */
#define HP_ADD         6   /* residual add of in0 and in1 */
#define HP_GAP         7   /* global average pool over (h,w) */
#define HP_SOFTMAX_CE  8   /* softmax cross-entropy head, K = classes; must be last */

/* ------------------------------------------------------ arithmetic modes */
#define HP_FP32  0         /* fp32 operands, fp32 accumulation */
#define HP_BF16  1         /* contraction operands rounded to bf16 (RNE), fp32 accumulation;
                              everything else, and all stored state, fp32 */

/* One layer of a stage.  Layers are listed in topological order; layer i's
 * output is value i and in0/in1 name the values a layer reads (-1 is the
 * stage input).  Parameters of the layers are concatenated in list order:
 *   HP_CONV  weight [K][R][S][C], then bias [K] if bias != 0
 *   HP_FC    weight [K][C] ([out][in]), then bias [K] if bias != 0
 *   HP_BN    gamma [C], then beta [C]
 * Fields a kind does not use are ignored. */
typedef struct hp_layer {
    int32_t kind;
    int32_t in0, in1;
    int32_t C, K;
    int32_t R, S;
    int32_t stride, pad;
    int32_t bias;
    float eps;
} hp_layer;

typedef struct hp_stage hp_stage;
typedef struct hp_ps hp_ps;
typedef struct hp_vw hp_vw;

/* ================================================================ stage */

/* Create a stage for minibatches of `batch` inputs of shape H x W x C (NHWC).
 * Allocates the activation stash, gradient buffers and workspaces on the
 * current HIP device; `stream` is a hipStream_t (NULL = default stream).
 * Errors: HP_ERR_ARG for an inconsistent layer list (shape mismatch, a loss
 * head that is not last, unknown kind), HP_ERR_NOMEM. */
int hp_stage_create(const hp_layer *layers, int n_layers, int batch, int H, int W, int C,
                    int dtype_mode, void *stream, hp_stage **out);
int hp_stage_destroy(hp_stage *st);

/* Number of fp32 parameters P of the stage. */
int hp_stage_param_count(const hp_stage *st, size_t *count);
/* Offset and length (in floats) of layer `layer`'s parameters in the flat
 * vector; both are 0 for a layer without parameters. */
int hp_stage_param_layout(const hp_stage *st, int layer, size_t *offset, size_t *count);
/* Per-image shape of layer `layer`'s output (layer -1: the stage output;
 * a loss head reports its logits).  dims = {H, W, C}; FC/GAP give {1, 1, C}. */
int hp_stage_output_shape(const hp_stage *st, int layer, int dims[3]);
/* Bytes of device memory the stage holds. */
int hp_stage_device_bytes(const hp_stage *st, size_t *bytes);
/* The same bytes by owner, for the model partitioner's memory model (HetPipe
 * Sec. 4, model partitioning): bytes[i] = buffers of layer i's value, its
 * gradient, its statistics and its bf16 copies; bytes[n_layers] = stage-level
 * buffers (contraction workspaces, bf16 weight copies, the input's bf16
 * copy).  n must be n_layers + 1; the entries sum to hp_stage_device_bytes. */
int hp_stage_layer_bytes(const hp_stage *st, size_t *bytes, int n);

/* Device timing of the stage's own kernels, for profiling.  While enabled,
 * every kernel the stage enqueues is bracketed by HIP events on the stage's
 * stream.  hp_stage_read_timing synchronises the stream, returns the summed
 * device time in milliseconds and the launch counts of two classes --
 * [0] contractions (implicit-GEMM conv / FC kernels and their split-K
 * reductions), [1] every other stage kernel -- and resets the sums. */
int hp_stage_set_timing(hp_stage *st, int enable);
int hp_stage_read_timing(hp_stage *st, double ms[2], int64_t launches[2]);
/* The same records per layer, for the model partitioner's per-layer profile
 * (HetPipe Sec. 4, model partitioning; Sec. 6, partitioning algorithm):
 * fwd_ms[i] / bwd_ms[i] receive the summed device time of the kernels that
 * the forward / backward pass enqueued for layer i (the weight gradient
 * included, whichever stream ran it); slot n_layers holds stage-level work
 * (the bf16 weight copies).  n must be n_layers + 1.  Synchronises the stream
 * and resets the records, like hp_stage_read_timing (either call consumes
 * them). */
int hp_stage_read_layer_timing(hp_stage *st, double *fwd_ms, double *bwd_ms, int n);

/* Forward pass of one minibatch (HetPipe Sec. 3: the layers of the stage in
 * order) at weights `w` (flat fp32, length P).  `x` is the stage input
 * [batch][H][W][C].  If the stage ends in HP_SOFTMAX_CE, `labels` (int32
 * [batch]) must be non-NULL, `loss` receives the mean cross-entropy (one
 * device float) and `y`, if non-NULL, the logits [batch][classes].  Otherwise
 * `labels` and `loss` must be NULL and `y` receives the stage output.
 * The activations needed by the backward pass are kept inside the stage. */
int hp_stage_forward(hp_stage *st, const float *w, const float *x, float *y,
                     const int32_t *labels, float *loss);

/* Backward pass of the minibatch whose forward ran last, at the same weights
 * `w` (Sec. 4: a minibatch's forward and backward use one weight version).
 * `dy` is the gradient at the stage output (NULL iff the stage ends in the
 * loss head).  `grad` (flat fp32, length P) is overwritten with the weight
 * gradient.  If `dx` is non-NULL it receives the gradient with respect to the
 * stage input; with dx == NULL the first layer's data gradient is skipped.
 * Errors: HP_ERR_STATE if no forward preceded or `w` differs from it. */
int hp_stage_backward(hp_stage *st, const float *w, const float *dy, float *dx, float *grad);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the
 * backward pass of hp_stage_backward -- same arguments, same kernels, same
 * results bit for bit -- with its workspaces (split-reduction partial tiles,
 * column-sum and batch-norm partials of the stage stream and of the
 * weight-gradient stream) taken from a static device array of the library,
 * HP_NOALLOC_SCRATCH_BYTES per device, instead of the stage's own.  Calls no
 * allocating routine.  Every call on one GPU shares that GPU's array, so
 * calls whose device work overlaps on one GPU (two stages on different
 * streams, or a call enqueued before the previous one has run) race: order
 * them on one stream.  Nothing in the array needs to start at zero: every
 * partial is written before it is read.  Must be called with the device
 * current on which the stage was created.
 * Errors: as hp_stage_backward; HP_ERR_ARG if the stage's workspaces exceed
 * HP_NOALLOC_SCRATCH_BYTES (the message gives both sizes); HP_ERR_STATE if
 * another device is current; HP_ERR_HIP if the array's device address cannot
 * be obtained. */
#define HP_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
int hp_stage_backward_noalloc(hp_stage *st, const float *w, const float *dy, float *dx,
                              float *grad);

/* Read-only device pointers to the buffers in which the stage holds layer
 * `layer`'s forward value and the gradient of the loss with respect to it, for
 * inspection (the layer-by-layer check of a real graph against a reference).
 * Both are [batch][H][W][C] fp32 (hp_stage_output_shape), owned by the stage
 * (or the caller, where noted), and valid until the next forward / backward
 * pass on the stage's stream.
 *   value: the layer's output from the last hp_stage_forward; NULL for the
 *          loss head and for a conv / FC / batch norm / add whose consumer
 *          ReLU it applies itself (its buffer holds the ReLU's output, which
 *          the ReLU layer reports).  Layer -1: the caller's stage input x.
 *   grad:  dL/d(value) from the last hp_stage_backward (the caller's dy for
 *          the last layer of a stage without loss head, the loss head's
 *          gradient for the logits); NULL where no buffer holds it after the
 *          pass: a ReLU whose mask its consumer applied, a batch norm that
 *          applies its consumer ReLU, an add whose buffer became its identity
 *          shortcut's gradient, a value no gradient reaches, or before any
 *          backward pass.  Layer -1: the caller's dx (NULL if none was asked).
 * Errors: HP_ERR_ARG for a NULL argument or a layer outside -1 .. n-1. */
int hp_stage_layer_buffers(const hp_stage *st, int layer, const float **value,
                           const float **grad);

/* ==================================================== parameter server */

/* Create the parameter server for N virtual workers with clock-distance
 * bound D (Sec. 5) holding w_g = copy of w0 (device pointer, P floats).
 * The server owns w_g.  c_g starts at 0. */
int hp_ps_create(size_t P, const float *w0, int N, int D, void *stream, hp_ps **out);
int hp_ps_destroy(hp_ps *ps);
/* Device pointer to w_g (read-only for the caller) and the global clock. */
int hp_ps_weights(const hp_ps *ps, const float **wg);
int hp_ps_clock(const hp_ps *ps, int *c_global);
/* Device timing of the WSP update kernels, for profiling.  While enabled,
 * every kernel enqueued by hp_wsp_local_update, hp_wsp_push_wave, hp_wsp_pull
 * and hp_wsp_wave_end of this server's virtual workers is bracketed by HIP
 * events on the server's stream.  hp_ps_read_timing synchronises the stream,
 * returns the summed device time in milliseconds and the launch counts of [0]
 * local updates whose minibatch starts a wave, [1] the other local updates,
 * [2] wave pushes, [3] pulls that copied w_g, [4] fused wave ends that pulled,
 * [5] fused wave ends that did not pull, and resets the sums. */
int hp_ps_set_timing(hp_ps *ps, int enable);
int hp_ps_read_timing(hp_ps *ps, double ms[6], int64_t launches[6]);

/* ======================================================= virtual worker */

/* Register virtual worker `id` (0 <= id < N) with the server.  The wave length
 * is W = s_local + 1 (Sec. 4: s_local = N_m - 1).  All W ring versions start
 * as copies of the server's current w_g (w_1 = ... = w_W = w_0). */
int hp_vw_create(hp_ps *ps, int id, int s_local, hp_vw **out);
int hp_vw_destroy(hp_vw *vw);

/* Starts the VW's next minibatch q = p + i + 1, where p minibatches have
 * completed and i (0 <= i < W) are in flight -- a VW runs up to N_m = W
 * minibatches concurrently in its pipeline (Sec. 4).  Returns the ring version
 * holding the local updates 1 .. q-W, a device pointer into the ring that
 * stays valid until minibatch q's own hp_wsp_local_update.  Minibatches
 * complete in the order they start.  Errors: HP_ERR_STATE if W minibatches are
 * already in flight, a completed wave has not been pushed yet, or its pull has
 * not succeeded. */
int hp_wsp_weights(hp_vw *vw, const float **w);

/* Momentum for this VW's local updates (an optimizer variant; the paper's
 * update is plain SGD, mu = 0): from now on hp_wsp_local_update computes
 *   v = mu * v + grad;  u = (-lr) * v
 * (heavy ball, no dampening, one rounding per operation) in place of
 * u = (-lr) * grad.  The velocity v (P floats, owned by the VW, local to it and
 * never pushed) is reset to zero by every call; mu = 0 restores plain SGD.
 * Errors: HP_ERR_ARG unless 0 <= mu < 1; HP_ERR_STATE while minibatches are
 * in flight. */
int hp_vw_set_momentum(hp_vw *vw, float mu);

/* Local update after the oldest in-flight minibatch q = p+1 completes (Sec. 4:
 * w_local = w_local + u_q, u_q = -lr * grad) and wave accumulation (Sec. 5:
 * u~ sums the wave's u_q).
 * Computes, element by element in fp32 without fused multiply-add,
 *   u = (-lr) * grad;  ring[(q-1) mod W] = ring[(q-2) mod W] + u;
 *   u~ = u (first minibatch of a wave) or u~ + u,
 * and advances p.  `grad` is caller-owned (P floats).
 * A wave end is settled before the next minibatch completes: after the update
 * that completes wave c, hp_wsp_push_wave and a successful hp_wsp_pull come
 * before the next hp_wsp_local_update.  The in-flight minibatches of wave c+1
 * may run their forward and backward passes meanwhile (Sec. 5: s_local
 * minibatches of the next wave proceed while the VW waits); only their
 * completion waits, so each includes exactly the updates 1 .. q-W.
 * Errors: HP_ERR_STATE if no minibatch is in flight, a completed wave has not
 * been pushed, or the pull after the push has not succeeded. */
int hp_wsp_local_update(hp_vw *vw, const float *grad, float lr);

/* Push at the end of wave c (Sec. 5): w_g = w_g + u~, the VW's local clock
 * becomes c+1 and c_g = min over VWs of their local clocks.  `ps` must be the
 * server the VW was created with.
 * Errors: HP_ERR_STATE unless the VW just completed a wave it has not pushed. */
int hp_wsp_push_wave(hp_vw *vw, hp_ps *ps);

/* Clock-bound gate after a push (Sec. 5, global staleness bound): the VW with
 * local clock c needs weights holding all VWs' waves 0 .. c-D-1.  If its last
 * pull already covers that, nothing happens (HP_OK).  Else if c_g >= c-D, w_g
 * is copied into the ring slot of the next wave's last minibatch, the pulled
 * clock becomes c_g (HP_OK).  Else HP_WOULD_BLOCK: the VW may not start a new
 * minibatch until a later hp_wsp_pull returns HP_OK, after other VWs pushed.
 * Never blocks the host thread.  A call with no pending gate returns HP_OK. */
int hp_wsp_pull(hp_vw *vw, hp_ps *ps);

/* Wave end in one call (Sec. 5, "Workings of WSP"): the local update of the
 * oldest in-flight minibatch q, which must complete a wave (q mod W = 0), the
 * push of that wave's aggregate u~ and the clock-bound gate, with the device
 * work of all three in one streaming pass over the parameters.  The results
 * -- ring, u~, w_g, clocks, version vectors, status -- are bit for bit those
 * of hp_wsp_local_update, hp_wsp_push_wave and hp_wsp_pull called in turn
 * (same fp32 operations, same order, no fused multiply-add); momentum, when
 * set, is applied as in hp_wsp_local_update.  When the gate opens at once
 * the new ring version is w_g itself and the newest version is not read
 * (24 bytes per parameter: read grad, u~, w_g; write u~, w_g, the ring slot).
 * Otherwise the slot gets the local version (28 bytes per parameter), and if
 * the gate is closed the call returns HP_WOULD_BLOCK exactly as hp_wsp_pull
 * does: retry hp_wsp_pull after other VWs pushed.  `grad` is caller-owned
 * (P floats); `ps` must be the VW's server.
 * Errors: HP_ERR_STATE if no minibatch is in flight, the oldest one does not
 * complete a wave, or an earlier wave end is unsettled. */
int hp_wsp_wave_end(hp_vw *vw, hp_ps *ps, const float *grad, float lr);

/* Host-side bookkeeping of a VW (exact integers). */
typedef struct hp_wsp_state {
    int64_t p;          /* minibatches completed */
    int32_t W;          /* wave length s_local + 1 */
    int32_t c;          /* local clock: waves pushed */
    int32_t g;          /* global clock reflected by the last pull */
    int32_t push_due;   /* a completed wave awaits hp_wsp_push_wave */
    int32_t gated;      /* a push happened and its pull has not succeeded */
    int32_t next_slot;  /* ring slot the next minibatch to start reads */
    int32_t n_vw;       /* N */
    int32_t in_flight;  /* minibatches started and not completed (0 .. W) */
} hp_wsp_state_t;
int hp_wsp_state(const hp_vw *vw, hp_wsp_state_t *out);

/* Version vector of the weights the next minibatch to start will read: V[n] = number
 * of minibatch updates of VW n contained in them (n < N).  `V` is host memory
 * of N int64 entries. */
int hp_wsp_version(const hp_vw *vw, int64_t *V);

/* Device pointers of the VW's ring and of u~ (P floats), owned by the VW; for
 * inspection.  Ring slot s starts at ring + s * slot_stride (slot_stride >= P,
 * a multiple of 64 floats so every slot is 256-byte aligned). */
int hp_wsp_buffers(const hp_vw *vw, const float **ring, size_t *slot_stride,
                   const float **utilde);

/* Description of the last error on the calling thread ("" if none). */
const char *hp_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* HETPIPE_H */
