/*
 * snn.h -- C ABI of libsnn.so: spiking-layer training on one MI355X (gfx950).
 *
 * The library computes one feed-forward spiking layer at a time, unrolled
 * over T time steps, and its backpropagation-through-time (BPTT) backward:
 *
 *   synapse   I[t,b,:] = W x[t,b,:] + bias     the "w x_t" term of eqs. (4)/(5);
 *             dense, or a 5x5 valid convolution followed by 2x2 max-pooling
 *             of the currents (the 5C12-MP2 / 5C64-MP2 layers of Table I)
 *   neuron    Leaky (eq. 4):  u_t = beta u_{t-1} + I_t - z_{t-1} thr
 *             Synaptic (eqs. 5-6): i_t = alpha i_{t-1} + I_t,
 *                                  u_t = beta u_{t-1} + i_t - z_{t-1} thr
 *             RLeaky (eq. 7): u_t = beta u_{t-1} + I_t + z_{t-1} (v - thr),
 *                             one recurrent weight v per neuron
 *             spike (eq. 3): z_t = 1 if u_t > thr (strict), else 0;
 *             initial state u = i = 0, no spike before the first step
 *   backward  the spike's derivative is replaced by the fast-sigmoid
 *             surrogate of eqs. (8)-(9) with slope k:
 *                 s_t = 1 / (1 + k |u_t - thr|)^2
 *             lam_t = g_t s_t + (beta - r thr s_t) lam_{t+1}  (r = 1 only for
 *             SNN_RESET_SURROGATE); Synaptic adds lami_t = lam_t + alpha lami_{t+1};
 *             RLeaky carries (beta + (v - r thr) s_t) lam_{t+1} and
 *             dL/dv = sum over t >= 1 and the batch of lam_t z_{t-1}.
 *             dL/dI_t = lam_t (Leaky, RLeaky) or lami_t (Synaptic), then
 *             dW = dI^T x, dbias = sum dI, dx = dI W.
 *   loss      on output spike counts c = sum_t z_t (rate-coded readout, the
 *             class is the neuron with most spikes, Sec. V): cross-entropy
 *             with c as logits (mean over the batch) or mean-squared error.
 *
 * Conventions for every entry point:
 *   - Tensor pointers are DEVICE pointers unless stated otherwise, row-major
 *     and contiguous, time-major [T, B, features] with features fastest.
 *     Every device pointer must be 16-byte aligned (SNN_ERR_ALIGN otherwise).
 *   - The caller owns and allocates every buffer, including `saved` and the
 *     workspace `ws` sized by the *_bytes queries.  The library allocates
 *     nothing, keeps no state between calls and is reentrant across streams.
 *   - Calls only enqueue work on `stream` (a hipStream_t; NULL = the null
 *     stream) and never synchronise the device.  Arguments are validated on
 *     the host before anything is launched; on error nothing is launched and
 *     outputs are untouched.  A failed launch returns SNN_ERR_HIP.
 *   - Outputs are overwritten, never accumulated into.
 *   - Arithmetic: contractions accumulate in fp32 with exact products.
 *     Spikes are exact in bf16 and fp16, an fp32 value is exactly three bf16
 *     parts and an fp16 value two, so contractions with a spike, fp16 or
 *     bf16 operand run on the 16-bit matrix cores as one pass per pair of
 *     parts (spike x fp32: three bf16 passes; spike x fp16: one fp16 pass),
 *     unless SNN_FLAG_FP32_MFMA is set; fp32 x fp32 runs on fp32 MFMA.
 *     Neuron state is fp32; loss reductions in fp64.
 *   - T == 0 or B == 0 is valid: no compute is launched, and outputs that
 *     are sums over an empty range (counts, grad_w, grad_b, grad_v) are set
 *     to 0.
 *     A loss over B == 0, K == 0 or P == 0 is rejected (SNN_ERR_SHAPE).
 */
#ifndef SNN_H
#define SNN_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SNN_ABI_VERSION 11

typedef enum snn_status {
    SNN_OK = 0,
    SNN_ERR_NULL = 1,        /* a required pointer is NULL */
    SNN_ERR_SHAPE = 2,       /* sizes negative, inconsistent or too large */
    SNN_ERR_DTYPE = 3,       /* dtype / format combination not supported */
    SNN_ERR_ALIGN = 4,       /* a device pointer is not 16-byte aligned */
    SNN_ERR_UNSUPPORTED = 5, /* a valid request the library does not implement */
    SNN_ERR_WORKSPACE = 6,   /* ws_bytes smaller than the query returned */
    SNN_ERR_HIP = 7          /* a kernel launch failed */
} snn_status;

/* element types */
#define SNN_F32 0
#define SNN_F16 1
#define SNN_BF16 2
#define SNN_U8 3 /* spikes stored as bytes 0 / 1 */
#define SNN_SPK_BITS 4 /* spikes packed 64 to a 64-bit word: neuron n of row
                          (t, b) is bit n % 64 of word n / 64 of that row's
                          n / 64 words (little-endian: bit n % 8 of byte
                          n / 8); an output type only, n_out a multiple of 64 */

/* neuron models */
#define SNN_LEAKY 0    /* eq. (4) */
#define SNN_SYNAPTIC 1 /* eqs. (5)-(6) */
#define SNN_RLEAKY 2   /* eq. (7): Leaky plus the neuron's own previous spike
                          through a recurrent weight v, one per neuron */

/* synapse kinds */
#define SNN_SYN_DENSE 0       /* x [T,B,n_in], w [n_out, n_in] */
#define SNN_SYN_CONV5_POOL2 1 /* x [T,B,c_in,h_in,w_in], w [c_out,c_in,5,5];
                                 currents [T,B,c_out,(h_in-4)/2,(w_in-4)/2] */
#define SNN_SYN_NONE 2        /* x already holds fp32 currents [T,B,n_out] */

/* gradient through the reset term -z_{t-1} thr */
#define SNN_RESET_DETACHED 0  /* reset treated as a constant in the backward */
#define SNN_RESET_SURROGATE 1 /* reset differentiated with the surrogate */

/* kinds of upstream gradient dL/dz for snn_layer_bwd / snn_neuron_bwd */
#define SNN_GRAD_FULL 0  /* g [T,B,n_out] fp32 */
#define SNN_GRAD_BCAST 1 /* g [B,n_out] fp32, the same for every t (a loss on
                            counts summed over T) */
#define SNN_GRAD_FOLD 2  /* g is the input gradient of a dense layer above with
                            n_up <= 16 outputs (a readout), computed inside the
                            reverse scan instead of being read:
                              g[t,b,n] = sum_{j < n_up} dcur_up[t,b,j] w_up[j,n]
                            in fp32 with j ascending (exact products), i.e.
                            the grad_x (dx = dI W) that layer's backward
                            would return.  It saves writing and re-reading
                            the [T,B,n_out] fp32 gradient.  Supported for
                            layers with n_out >= 64 (SNN_ERR_UNSUPPORTED
                            otherwise). */

/* descriptor flags */
#define SNN_FLAG_FP32_MFMA 1 /* run every contraction on fp32 MFMA instead of
                                exact multi-part passes on the 16-bit matrix
                                cores (an fp32 operand split into hi + mid +
                                lo bf16 parts, fp16 into two bf16 parts or
                                kept as fp16; every product exact, fp32
                                accumulate) */

/* losses on spike counts */
#define SNN_LOSS_CE_COUNT 0  /* labels int32 [B] in [0,K) */
#define SNN_LOSS_MSE_COUNT 1 /* targets fp32 [B,K] */

typedef struct snn_layer_desc {
    int32_t T, B;           /* time steps, batch */
    int32_t synapse;        /* SNN_SYN_* */
    int32_t neuron;         /* SNN_LEAKY | SNN_SYNAPTIC | SNN_RLEAKY */
    int32_t n_in, n_out;    /* features per (t,b) of x and of the output;
                               conv: c_in*h_in*w_in and c_out*hp*wp;
                               SNN_SYN_NONE: n_in == n_out */
    int32_t c_in, h_in, w_in, c_out; /* conv geometry, else ignored */
    int32_t in_dtype;       /* x: SNN_U8 spikes, SNN_F32 (also SYN_NONE), SNN_F16,
                               or SNN_BF16 (dense layers with SNN_F32 weights:
                               spikes in the operand type of the three-plane
                               contractions, no widening per call) */
    int32_t w_dtype;        /* w: SNN_F32 | SNN_F16 */
    int32_t out_dtype;      /* spikes written as SNN_U8 | SNN_F16 (0.0 / 1.0) |
                               SNN_SPK_BITS ([T,B,n_out / 8] bytes; n_out a
                               multiple of 64, else SNN_ERR_SHAPE) */
    int32_t grad_dtype;     /* dL/dI handed to the weight / input gradient
                               contractions: SNN_F32 | SNN_BF16 | SNN_F16.
                               SNN_F16 holds dL/dI * S, S a power of two
                               chosen per backward call so that every value
                               stays below 2^15 (see snn_neuron_bwd); not for
                               SNN_RLEAKY */
    int32_t reset_grad;     /* SNN_RESET_DETACHED | SNN_RESET_SURROGATE */
    int32_t flags;          /* 0 or SNN_FLAG_FP32_MFMA */
    float beta;             /* membrane decay, eqs. (4)/(6) */
    float alpha;            /* synaptic decay, eq. (5); ignored for Leaky, RLeaky */
    float threshold;        /* u_thr */
    float slope;            /* surrogate slope k (k = 1 is eq. (9) as printed) */
} snn_layer_desc;

typedef struct snn_grad_in {
    int32_t kind;          /* SNN_GRAD_FULL | SNN_GRAD_BCAST | SNN_GRAD_FOLD */
    int32_t n_up;          /* SNN_GRAD_FOLD: outputs of the layer above, 1..16
                              (SNN_ERR_SHAPE otherwise); must be 0 for the
                              other kinds (SNN_ERR_UNSUPPORTED) */
    const float *g;        /* FULL / BCAST: dL/dz of this layer's output
                              spikes, fp32; ignored for FOLD */
    const void *dcur_up;   /* FOLD: dL/dI of the layer above, [T,B,n_up] of
                              dcur_up_dtype (its snn_neuron_bwd output) */
    const void *w_up;      /* FOLD: weights of the layer above, [n_up, n_out]
                              of w_up_dtype */
    int32_t dcur_up_dtype; /* FOLD: SNN_F32 | SNN_BF16 | SNN_F16 */
    int32_t w_up_dtype;    /* FOLD: SNN_F32 | SNN_F16 */
} snn_grad_in;

int snn_abi_version(void);
const char *snn_status_str(snn_status s);

/* Bytes of the forward-to-backward state (BPTT keeps O(n T) state, Sec.
 * II-B).  The backward needs the membrane u_t of every step (the surrogate
 * of eq. (9) depends on nothing else); instead of u_t the state holds the
 * currents and the neuron state every ckpt_interval steps, from which the
 * reverse scan recomputes u_t chunk by chunk (bit-identical: the same fp32
 * operations as the forward). */
size_t snn_layer_saved_bytes(const snn_layer_desc *d);

/* Where each part of the saved state lies inside the snn_layer_saved_bytes
 * buffer (byte offsets, each a multiple of 256):
 *   cur    fp32 currents I [T,B,n_out] of the synapse, as the forward scan
 *          read them (0 bytes for SNN_SYN_NONE: the layer's x holds them)
 *   ckpt   checkpoints: fp32 [ckpt_planes][ckpt_count][B*n_out]; slot c
 *          (0 <= c < ckpt_count = (T - 1) / ckpt_interval) holds the state
 *          after step (c + 1) * ckpt_interval - 1 (0-based): plane 0 the
 *          membrane u, plane 1 (SNN_SYNAPTIC only) the synaptic current i
 *   pool   conv only: u8 [T,B,n_out] 2x2 pool selection 0..3 (row-major in
 *          the window, first maximum wins); 0 bytes otherwise
 * The stage calls take these parts as separate pointers. */
typedef struct snn_saved_layout {
    size_t bytes;               /* == snn_layer_saved_bytes */
    size_t cur_offset, cur_bytes;
    size_t ckpt_offset, ckpt_bytes;
    size_t pool_offset, pool_bytes;
    int32_t ckpt_interval;      /* steps between checkpoints */
    int32_t ckpt_count;         /* checkpoints per plane */
    int32_t ckpt_planes;        /* 1, or 2 for SNN_SYNAPTIC */
    int32_t reserved;
} snn_saved_layout;
/* SNN_ERR_NULL for a NULL out; the descriptor's errors otherwise. */
snn_status snn_layer_saved_layout(const snn_layer_desc *d, snn_saved_layout *out);

/* Scratch bytes needed by snn_layer_fwd / snn_layer_bwd and the stage calls
 * below (the maximum over all of them).  0 is a valid answer. */
size_t snn_layer_workspace_bytes(const snn_layer_desc *d);

/* Forward of one layer (synapse, then the neuron scan over all T; eqs.
 * (3)-(7) after the w x_t contraction).
 *   x       [T,B,n_in] of d->in_dtype
 *   w       weights of d->w_dtype (NULL iff SNN_SYN_NONE)
 *   bias    fp32 [n_out] dense / [c_out] conv, or NULL for no bias
 *   v       fp32 [n_out] recurrent weights of SNN_RLEAKY (one per output
 *           neuron, the same for every sample); required for SNN_RLEAKY
 *           (SNN_ERR_NULL), ignored for the other neurons
 *   spk_out [T,B,n_out] spikes of d->out_dtype
 *   saved   snn_layer_saved_bytes(d) bytes, kept for snn_layer_bwd
 *   counts  fp32 [B,n_out] spike counts sum_t z_t, or NULL
 *   ws      snn_layer_workspace_bytes(d) bytes (may be NULL if 0) */
snn_status snn_layer_fwd(const snn_layer_desc *d, const void *x, const void *w,
                         const float *bias, const float *v, void *spk_out, void *saved,
                         float *counts, void *ws, size_t ws_bytes, hipStream_t stream);

/* Backward of one layer (reverse-time neuron scan, then the synapse; BPTT
 * with the surrogate of eqs. (8)-(9)).
 *   grad    upstream dL/dz of this layer's spikes
 *   x, w, v the forward's inputs (x required for SNN_SYN_NONE: its currents);
 *           saved: the forward's saved state
 *   grad_w  dL/dw (layout of w, fp32), NULL to skip; must be NULL for SYN_NONE
 *   grad_b  dL/dbias fp32, NULL to skip
 *   grad_v  dL/dv fp32 [n_out] of SNN_RLEAKY, NULL to skip; must be NULL for
 *           the other neurons (SNN_ERR_SHAPE)
 *   grad_x  dL/dx fp32 [T,B,n_in] (the g of the layer below), NULL to skip;
 *           for SNN_SYN_NONE this is dL/dI and is required */
snn_status snn_layer_bwd(const snn_layer_desc *d, const snn_grad_in *grad, const void *x,
                         const void *w, const float *v, const void *saved, float *grad_w,
                         float *grad_b, float *grad_v, float *grad_x, void *ws,
                         size_t ws_bytes, hipStream_t stream);

/* Loss on spike counts and its gradient dL/dcounts (which is dL/dz_t for
 * every t, since dc/dz_t = 1).  K classes, P >= 1 output neurons per class:
 * counts and grad_counts are [B, K*P]; with P > 1 (a population code, Sec. V)
 * class k's count c_k is the sum of neurons kP .. kP+P-1, and each neuron of
 * a population receives its class's gradient.  `loss` is a device fp32
 * scalar.  Over the class counts c [B,K]:
 * CE: L = mean_b (logsumexp(c_b) - c_b[y_b]),  g = (softmax(c_b) - onehot)/B.
 * MSE: L = mean (c - y)^2 (targets [B,K]),    g = 2 (c - y) / (B K). */
size_t snn_loss_workspace_bytes(int32_t kind, int32_t B, int32_t K);
snn_status snn_loss(int32_t kind, int32_t B, int32_t K, int32_t P, const float *counts,
                    const int32_t *labels, const float *targets, float *loss,
                    float *grad_counts, void *ws, size_t ws_bytes, hipStream_t stream);

/* The same loss for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * no workspace argument; the partial sums live in a 1 MiB device array the
 * library holds on every device it runs on (until the process ends).  Sizes
 * whose snn_loss_workspace_bytes exceeds 1 MiB (cross-entropy over more than
 * 131072 rows) are rejected with SNN_ERR_WORKSPACE; the other checks and
 * errors are those of snn_loss.  Nothing is allocated and no state carries
 * over between calls, but every call on one device shares that array: calls
 * that overlap on one device (two streams, two host threads) race. */
snn_status snn_loss_noalloc(int32_t kind, int32_t B, int32_t K, int32_t P, const float *counts,
                            const int32_t *labels, const float *targets, float *loss,
                            float *grad_counts, hipStream_t stream);

/* ---- whole step of a small two-layer network in one launch -----------------
 * Forward, loss and BPTT backward of a dense hidden layer (spike input x
 * [T,B,n_in] u8 0 / 1, a nonzero byte counting as 1; fp32 weights) and a
 * dense readout whose spike counts feed the loss, as one kernel: for small batches (Sec. IV's small-batch
 * results), where the step as separate calls is a chain of launch
 * latencies.  The arithmetic is that of snn_layer_fwd / snn_loss /
 * snn_layer_bwd on the same network with the readout's input gradient folded
 * into the hidden layer's reverse scan: exact products of the spikes with
 * the fp32 weights' three bf16 parts, fp32 accumulation (in another order
 * than the layer calls, so a current may differ in its last bits), the same
 * scans, adjoints and loss.  Workgroups own hidden neurons; grid-wide
 * barriers separate packing the input to bits, the hidden forward, the
 * readout with the loss, and the hidden backward.  The grid is at most one
 * workgroup per compute unit (resident at once on an otherwise idle device);
 * each barrier wait polls at most wait_limit times (0: a default of about
 * 0.1 s or more), and a workgroup that gives up writes 1 to *status and
 * skips the rest of the step, so the launch ends whatever happens (the
 * outputs are then undefined; so it goes when another kernel holds compute
 * units meanwhile).  *status is 0 after a step that
 * completed.  The barrier counters are device state of the library, clear
 * after every launch: calls that overlap on one device must not be made. */
typedef struct snn_fused_desc {
    snn_layer_desc hidden;   /* SNN_SYN_DENSE, in_dtype SNN_U8, w_dtype SNN_F32,
                                SNN_LEAKY or SNN_SYNAPTIC, n_in and n_out
                                multiples of 8 */
    snn_layer_desc readout;  /* SNN_SYN_DENSE, n_in = hidden.n_out, n_out <= 16,
                                w_dtype SNN_F32, same T (1..32) and B (>= 1),
                                SNN_LEAKY or SNN_SYNAPTIC */
    int32_t loss_kind;       /* SNN_LOSS_CE_COUNT | SNN_LOSS_MSE_COUNT */
    int32_t pop;             /* population size P, readout.n_out = K * P */
    uint32_t wait_limit;     /* polls per barrier wait before giving up; 0: default */
    int32_t reserved;        /* 0 */
} snn_fused_desc;

/* SNN_OK if snn_fused_step runs this network on the current device, else the
 * reason: SNN_ERR_UNSUPPORTED (layer kinds, neurons, sizes above, too many
 * hidden neurons or too large T*B for one co-resident grid with its state in
 * LDS), SNN_ERR_DTYPE, SNN_ERR_SHAPE, or the layer descriptors' own errors. */
snn_status snn_fused_step_check(const snn_fused_desc *d);
size_t snn_fused_step_workspace_bytes(const snn_fused_desc *d);

/* x [T,B,n_in] u8; w0 [n_hid,n_in], b0 [n_hid] (nullable), w1 [n_out,n_hid],
 * b1 [n_out] (nullable), fp32.  labels int32 [B] (cross-entropy) or targets
 * fp32 [B,K] (MSE).  Outputs (each nullable except status): loss (fp32 [1],
 * the batch mean as snn_loss), counts [B,n_out] (readout spike counts),
 * spk_hidden u8 [T,B,n_hid] (the hidden layer's spikes), grad_w0, grad_b0,
 * grad_w1, grad_b1 (fp32, shapes of the parameters); status int32 [1] on the
 * device.  All device pointers 16-byte aligned. */
snn_status snn_fused_step(const snn_fused_desc *d, const uint8_t *x, const float *w0,
                          const float *b0, const float *w1, const float *b1,
                          const int32_t *labels, const float *targets, float *loss,
                          float *counts, uint8_t *spk_hidden, float *grad_w0, float *grad_b0,
                          float *grad_w1, float *grad_b1, int32_t *status, void *ws,
                          size_t ws_bytes, hipStream_t stream);

/* ---- weight update ---------------------------------------------------------
 * AdamW, the optimizer the paper trains every network with (Sec. IV): for
 * each parameter tensor, elementwise, with step t >= 1,
 *     theta <- theta (1 - lr wd)
 *     m <- beta1 m + (1 - beta1) g,      v <- beta2 v + (1 - beta2) g^2
 *     theta <- theta - lr (m / (1 - beta1^t)) / (sqrt(v / (1 - beta2^t)) + eps)
 * (Adam's bias-corrected moments, weight decay decoupled from the gradient).
 * All tensors of a call are updated by one fused pass (one kernel launch per
 * 16 non-empty tensors).  param, m, v are fp32 and updated in place (param is
 * the fp32 master copy); grad is fp32 (the grad_w / grad_b / grad_v of the
 * backward).  param_half, if not NULL, receives the updated param rounded to
 * fp16 (nearest even): the weights an SNN_F16 layer contracts with.  The
 * arrays of one tensor must not overlap each other or another tensor's. */
typedef struct snn_adamw_tensor {
    float *param;        /* fp32 [n], in place */
    const float *grad;   /* fp32 [n] */
    float *m;            /* fp32 [n] first moment, in place (zeros before step 1) */
    float *v;            /* fp32 [n] second moment, in place (zeros before step 1) */
    void *param_half;    /* fp16 [n] copy of the updated param, or NULL */
    int64_t n;           /* elements, 0 <= n <= 2^36 (n = 0: skipped) */
} snn_adamw_tensor;

typedef struct snn_adamw_hparams {
    float lr;            /* >= 0 */
    float beta1, beta2;  /* in [0, 1) */
    float eps;           /* >= 0 */
    float weight_decay;  /* >= 0 */
    int32_t step;        /* t >= 1: the t-th update of these moments */
} snn_adamw_hparams;

/* tensors: HOST array of `count` descriptors (count >= 0; NULL iff 0) whose
 * pointers are device pointers; hp: host pointer.  SNN_ERR_NULL for a
 * missing pointer of a non-empty tensor, SNN_ERR_SHAPE for bad sizes or
 * hyper-parameters (non-finite, out of range, step < 1). */
snn_status snn_adamw(const snn_adamw_tensor *tensors, int32_t count,
                     const snn_adamw_hparams *hp, hipStream_t stream);

/* ---- stage calls: the two halves of snn_layer_fwd / snn_layer_bwd -------
 * snn_layer_fwd == snn_synapse_fwd(cur = saved) + snn_neuron_fwd(cur = saved,
 * saved_u = saved); snn_layer_bwd == snn_neuron_bwd + snn_synapse_bwd.  They
 * let a caller time the contraction and the scan separately (the paper's
 * split of time between synaptic and neuron work, Sec. IV) and check each
 * stage on its own. */

/* Synapse forward (the w x_t term of eqs. (4)/(5); Table I's conv + pool):
 * currents I [T,B,n_out] fp32.  pool_arg: conv only, u8 [T,B,n_out] pool
 * selection 0..3 (row-major in the 2x2 window, first maximum wins). */
snn_status snn_synapse_fwd(const snn_layer_desc *d, const void *x, const void *w,
                           const float *bias, float *cur, uint8_t *pool_arg, void *ws,
                           size_t ws_bytes, hipStream_t stream);

/* Neuron scan over T (eqs. 3-7): spikes spk_out [T,B,n_out] of
 * d->out_dtype, counts (nullable) [B,n_out], and the checkpoints ckpt laid
 * out as the ckpt part of snn_saved_layout (required when ckpt_count > 0).
 * u_out (nullable): the membrane u_t of every step, fp32 [T,B,n_out]; it may
 * be the same pointer as cur (in place), any other overlap is undefined.
 * v as in snn_layer_fwd. */
snn_status snn_neuron_fwd(const snn_layer_desc *d, const float *cur, const float *v,
                          void *spk_out, float *ckpt, float *u_out, float *counts,
                          hipStream_t stream);

/* Reverse-time scan (eqs. 8-9 through the recursion of the header above)
 * from the forward's currents cur [T,B,n_out] fp32 and checkpoints ckpt (as
 * written by snn_neuron_fwd on the same currents; u_t is recomputed):
 * dcur = dL/dI [T,B,n_out] of d->grad_dtype, grad_b (nullable) = sum of dL/dI
 * over t, b (and pooled positions), and grad_v (nullable, SNN_RLEAKY only) as
 * in snn_layer_bwd.
 * dcur_scale: with grad_dtype SNN_F16, a device fp32 scalar (required) that
 * receives the power of two S; dcur then holds fp16(dL/dI * S).  S is the
 * largest power of two with G F S <= 2^15, where G bounds |dL/dz| over the
 * upstream gradient (max |g|; for SNN_GRAD_FOLD max over (t,b) of
 * sum_j |dcur_up| times max |w_up|, a device reduction) and F bounds the
 * growth of the recursion, sum_{k<T} c^k with c = max(|beta|, |beta - r thr|)
 * (times sum_{k<T} |alpha|^k for SNN_SYNAPTIC); so no value overflows fp16
 * and the rounding of each value is relative 2^-11 above 2^-14 / S.
 * SNN_F16 is rejected for SNN_RLEAKY and where F exceeds 1e30
 * (SNN_ERR_UNSUPPORTED).  Ignored (may be NULL) for the other dtypes.
 * dcur_t (nullable, dense layers only, snn_layer_dcur_t_bytes(d) bytes): the
 * same dL/dI written as the weight gradient's operand, so that
 * snn_synapse_bwd needs no transpose or split, in the layout
 * snn_layer_dcur_t_layout(d) names: SNN_DCUR_T_TRANSPOSED, 16-bit
 * [P][n_out][B*T], row n holding neuron n of every sample, column b*T + t
 * (sample-major), P = 3 exact bf16 parts (hi, mid, lo: hi = bf16(x), mid =
 * bf16(x - hi), lo = bf16(x - hi - mid)) for SNN_F32, else 1 plane of
 * d->grad_dtype (fp16 scaled as dcur); SNN_DCUR_T_PLANES, the same three
 * parts of an fp32 dL/dI as [3][T*B][n_out].  dcur may be NULL when dcur_t
 * is given. */
snn_status snn_neuron_bwd(const snn_layer_desc *d, const snn_grad_in *grad, const float *v,
                          const float *cur, const float *ckpt, void *dcur, void *dcur_t,
                          float *dcur_scale, float *grad_b, float *grad_v, void *ws,
                          size_t ws_bytes, hipStream_t stream);

/* Synapse backward from dcur (of d->grad_dtype): grad_w and/or grad_x
 * (dW = dI^T x and dx = dI W, BPTT through the w x_t term of eqs. (4)/(5)).
 * dcur_t (nullable): the operand snn_neuron_bwd wrote; the weight gradient
 * contracts it instead of transposing or splitting dcur (used when
 * snn_layer_dcur_t_bytes(d) > 0).  dcur may then be NULL unless grad_x is
 * requested.  dcur_scale: for SNN_F16, the scale snn_neuron_bwd wrote
 * (required); the contractions divide it out.  Ignored for the other
 * dtypes. */
snn_status snn_synapse_bwd(const snn_layer_desc *d, const void *dcur, const void *dcur_t,
                           const float *dcur_scale, const uint8_t *pool_arg, const void *x,
                           const void *w, float *grad_w, float *grad_x, void *ws,
                           size_t ws_bytes, hipStream_t stream);

/* Bytes of the transposed dL/dI operand (dcur_t of snn_neuron_bwd /
 * snn_synapse_bwd), or 0 when the layer's weight gradient does not take it
 * (conv layers, layers with at most 16 outputs, small products, and large
 * products of a 16-bit dL/dI, which read dL/dI and x in their own
 * layouts). */
size_t snn_layer_dcur_t_bytes(const snn_layer_desc *d);

/* Layout of the dcur_t operand snn_neuron_bwd writes for this layer (-1 for
 * an invalid descriptor):
 * SNN_DCUR_T_TRANSPOSED: 16-bit [P][n_out][B*T] as described at
 *   snn_neuron_bwd (P = 3 exact bf16 parts for SNN_F32, else 1);
 * SNN_DCUR_T_PLANES: an fp32 dL/dI as its three exact bf16 parts (hi, mid,
 *   lo, as above) in dL/dI's own layout, [3][T*B][n_out], for a weight
 *   gradient that reads dL/dI untransposed (large dense fp32 layers whose
 *   n_out and n_in are multiples of 8).  snn_layer_bwd has the scan write
 *   these planes in place of the fp32 dL/dI when the layer has no input
 *   gradient to compute. */
#define SNN_DCUR_T_TRANSPOSED 1
#define SNN_DCUR_T_PLANES 2
int32_t snn_layer_dcur_t_layout(const snn_layer_desc *d);

#ifdef __cplusplus
}
#endif

#endif /* SNN_H */
