// Internal launch interface of libsnn.so (not part of the public ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "snn.h"

namespace snn {

constexpr size_t kAlign = 256;  // workspace sub-buffers start on 256-byte boundaries

inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

constexpr int kXcds = 8;  // MI355X: 8 accelerator complex dies, one L2 each

// Linear workgroup id renumbered so that the workgroups the dispatcher sends
// to one XCD (ids congruent mod 8) cover one contiguous range of work items.
// A bijection on [0, gridDim.x * gridDim.y * gridDim.z).
__device__ inline int xcd_local_item() {
    const int lin = blockIdx.x + gridDim.x * (blockIdx.y + gridDim.y * blockIdx.z);
    const int total = gridDim.x * gridDim.y * gridDim.z;
    const int xcd = lin % kXcds, idx = lin / kXcds;
    const int per = total / kXcds, rem = total % kXcds;
    return xcd < rem ? xcd * (per + 1) + idx : rem * (per + 1) + (xcd - rem) * per + idx;
}

// Internal operand type: an fp32 array held exactly as three bf16 planes
// (hi, mid, lo), the plane stride given by GemmArgs::a_ps / b_ps.
constexpr int kPlanes3 = 64;

inline size_t dtype_bytes(int dt) {
    switch (dt) {
        case kPlanes3: return 6;
        case SNN_F32: return 4;
        case SNN_F16: return 2;
        case SNN_BF16: return 2;
        case SNN_U8: return 1;
        default: return 0;
    }
}

// Compute units of the current device (cached per device).
int device_cus();

// ---- neuron scans (scan.hip) ---------------------------------------------
// The forward saves the neuron state every kCheckpointInterval steps; the
// reverse scan recomputes each chunk from it and the currents.  Checkpoint c
// (0 <= c < neuron_ckpt_count(T)) is the state after step (c + 1) K - 1:
// ckpt[c][C] holds u and, for SNN_SYNAPTIC, ckpt[count + c][C] holds i.
constexpr int kCheckpointInterval = 16;
int64_t neuron_ckpt_count(int T);
// Forward: C = B * N independent columns, time-major [T, C]; vrec [N] holds
// the recurrent weights of SNN_RLEAKY (column c is neuron c % N), else unused.
// u_out (nullable) receives the membrane of every step.
hipError_t launch_neuron_fwd(int neuron, int T, int64_t C, int64_t N, float alpha, float beta,
                             float thr, const float *vrec, const float *cur, void *spk,
                             int out_dtype, float *u_out, float *ckpt, float *counts,
                             hipStream_t s);

// Upstream gradient of the reverse scan: g [T, C] (SNN_GRAD_FULL), g [C] for
// every t (SNN_GRAD_BCAST), or, for SNN_GRAD_FOLD, computed in the scan as
// g[t, b, n] = sum_{j < nup} dup[t, b, j] wup[j, n] (nup <= 16; layers with
// N >= 64 only, see neuron_fold_supported).
struct BwdGrad {
    int mode;
    const float *g;
    const void *dup, *wup;
    int nup, dt_up, dt_w;
};
bool neuron_fold_supported(int64_t N);

// Backward: writes dcur [T, C] (grad_dtype), colsum [C] = sum_t dL/dI (fp32,
// may be NULL) and, for SNN_RLEAKY, dvcol [C] = sum_t lam_{t+1} z_t (fp32,
// may be NULL).  C = B * N.  An SNN_F16 dcur holds dL/dI * S with the power
// of two S read from dscale[0] (launch_grad_scale writes it).
// dcur_t (nullable): dL/dI also written as the weight gradient's operand,
// [P][N][B*T] 16-bit (P = 3 exact bf16 parts of fp32, else 1), K index b*T + t;
// with dcur_t_planes (fp32 only) instead the three exact bf16 parts in dcur's
// own layout, [3][T][C].  dcur may be NULL when dcur_t is given.
hipError_t launch_neuron_bwd(int neuron, int reset_surrogate, int T, int64_t C, int64_t N,
                             float alpha, float beta, float thr, float slope, const float *vrec,
                             const float *cur, const float *ckpt, const BwdGrad &grad, int B,
                             void *dcur, void *dcur_t, bool dcur_t_planes, int grad_dtype,
                             const float *dscale, float *colsum, float *dvcol, hipStream_t s);
// scale[0] = S = 2^e, the largest power of two with G * growth * S <= 2^15,
// G a bound on |g| over the upstream gradient (device reduction into
// `scratch`, grad_scale_workspace_bytes()); growth bounds |dL/dI| / G.
size_t grad_scale_workspace_bytes();
hipError_t launch_grad_scale(int T, int64_t C, const BwdGrad &grad, int B, double growth,
                             float *scale, float *scratch, hipStream_t s);

// p[0..n) = 0 with a kernel (safe inside captured graphs)
hipError_t launch_fill_zero(float *p, int64_t n, hipStream_t s);

// db[f] = sum_b sum_p colsum[b*F*P + f*P + p]  (fixed order)
hipError_t launch_bias_reduce(int B, int F, int P, const float *colsum, float *db, hipStream_t s);

// ---- GEMM (gemm.hip) -------------------------------------------------------
// C[M,N] = sum_k A(m,k) * B(n,k) (+ bias[n]).  A(m,k) = A[m*lda + k] when a_kc
// (K contiguous) else A[k*lda + m]; likewise B.  Element types SNN_F32, SNN_F16,
// SNN_BF16 or SNN_U8; products accumulate in fp32.  Split-K partials go to ws.
struct GemmArgs {
    int M, N, K;
    const void *A;
    int64_t lda;
    int a_dtype;
    bool a_kc;
    const void *B;
    int64_t ldb;
    int b_dtype;
    bool b_kc;
    float *C;
    int64_t ldc;
    const float *bias;  // [N] or NULL
    bool allow_split;   // may run on 16-bit MFMA as exact multi-part passes
    int64_t a_ps = 0, b_ps = 0;  // plane strides (elements) of kPlanes3 operands
    // 2x2 max-pool epilogue (convolution forward): rows m = 4 q + d are the
    // four window positions of pooled cell q.  A contraction that can pool
    // its own output (one pass over K, no split) writes the first maximum
    // (C + bias) to pool_cur[(q / pool_hw) * N + n][q % pool_hw] and its d to
    // pool_arg instead of C, and sets *pooled; otherwise C is written.
    int pool_hw = 0;
    float *pool_cur = nullptr;
    uint8_t *pool_arg = nullptr;
    bool *pooled = nullptr;
    // C is divided by c_div[0] (a device power of two, the scale of an fp16
    // dL/dI operand); NULL: no scaling
    const float *c_div = nullptr;
};
size_t gemm_workspace_bytes(int M, int N, int K, int a_dtype, int b_dtype, bool a_kc,
                            bool b_kc, bool allow_split);
hipError_t launch_gemm(const GemmArgs &g, void *ws, size_t ws_bytes, hipStream_t s);
// C[m,n] = sum_{z<S} P[z][m][n] / c_div[0] (+ bias[n]), fixed order (c_div may be NULL)
hipError_t launch_splitk_reduce(int M, int N, int S, const float *P, float *C, int64_t ldc,
                                const float *bias, hipStream_t s, const float *c_div = nullptr);
// C[m,n] /= c_div[0] for m < M, n < N
hipError_t launch_divide(int M, int N, float *C, int64_t ldc, const float *c_div, hipStream_t s);

// ---- 16-bit matrix cores, exact products (gemm_mfma16.hip) ---------------------
bool gemm16_applies(const GemmArgs &g);
size_t gemm16_workspace_bytes(const GemmArgs &g);
hipError_t launch_gemm16(const GemmArgs &g, void *ws, size_t ws_bytes, hipStream_t s);
int gemm16_passes(const GemmArgs &g);  // MFMA passes per product, 0 if not applicable
// dst[p][rows][ldp] = part p (hi, mid, lo) of the exact three-bf16 split of
// src[r * ld + k], k < K; columns K .. ldp - 1 are 0
hipError_t launch_split_planes(const float *src, int64_t ld, int rows, int K, int ldp,
                               uint16_t *dst, hipStream_t s);
// ---- contractions of layers with few outputs (skinny.hip) --------------------
// short contraction: K <= 16, A K-contiguous, B N-contiguous
bool short_k_applies(const GemmArgs &g);
hipError_t launch_short_k(const GemmArgs &g, hipStream_t s);
// few rows: M <= 16, A and B M/N-contiguous (the weight gradient of such a layer)
bool few_rows_applies(const GemmArgs &g);
size_t few_rows_workspace_bytes(const GemmArgs &g);
hipError_t launch_few_rows(const GemmArgs &g, void *ws, size_t ws_bytes, hipStream_t s);

// forward of a layer with at most 16 outputs and a long contraction: A
// spikes (bytes) or fp16, W fp32 or fp16, both K-contiguous; 16-bit MFMA with
// exact products (needs allow_split)
bool narrow_fwd_applies(const GemmArgs &g);
hipError_t launch_narrow_fwd(const GemmArgs &g, hipStream_t s);

// ---- large single-part contractions, asynchronous LDS pipeline (gemm_async.hip)
bool gemm_async_applies(const GemmArgs &g);
size_t gemm_async_workspace_bytes(const GemmArgs &g);
hipError_t launch_gemm_async(const GemmArgs &g, void *ws, size_t ws_bytes, hipStream_t s);

// dst[c*ld_dst + k] = src[row(k)*ld_src + c] for k < rows, c < cols, with
// row(k) = k, or, when perm_T > 0, row(k) = (k % perm_T) * (rows / perm_T) +
// k / perm_T (a [T][B] row index read in the order k = b*T + t); to_planes
// writes an fp32 source as three bf16 planes `plane` elements apart.
hipError_t launch_transpose(int rows, int cols, const void *src, int64_t ld_src, int elem_bytes,
                            void *dst, int64_t ld_dst, bool to_planes, int64_t plane,
                            hipStream_t s, int perm_T = 0);

// ---- losses (loss.hip) -----------------------------------------------------
size_t loss_workspace_bytes(int kind, int B, int K);
// counts / grad [B, K*P] (P neurons per class), targets [B, K]
hipError_t launch_loss(int kind, int B, int K, int P, const float *counts,
                       const int32_t *labels, const float *targets, float *loss, float *grad,
                       void *ws, hipStream_t s);
// The loss's scratch held by the library (a static device array, 1 MiB per
// device): its address on the current device, looked up on first use.
constexpr size_t kLossScratchBytes = (size_t)1 << 20;
hipError_t loss_static_scratch(void **ptr);

// ---- AdamW weight update (optim.hip) -------------------------------------------
// per-step coefficients, computed on the host in double
struct AdamwCoef {
    float decay;            // 1 - lr * weight_decay
    float beta1, one_minus_beta1, beta2, one_minus_beta2;
    float step_size;        // lr / (1 - beta1^t)
    float inv_sqrt_bc2;     // 1 / sqrt(1 - beta2^t)
    float eps;
};
constexpr int kAdamwMaxTensors = 16;  // tensors per launch (kernel arguments by value)
int64_t adamw_blocks(int64_t n);
// tensors: host array of the caller's descriptors (validated)
hipError_t launch_adamw(const snn_adamw_tensor *t, int count, const AdamwCoef &c, hipStream_t s);

// ---- convolution + pool (conv.hip) -------------------------------------------
struct ConvGeom {
    int NB;   // T * B images
    int Ci, H, W, Co;
    int Ho, Wo, Hp, Wp;  // conv output and pooled sizes
};
// every tensor and GEMM buffer of the layer indexes in int32
bool conv_fits_int32(const ConvGeom &g);
size_t conv_fwd_workspace_bytes(const ConvGeom &g, int in_dtype, bool allow_split);
size_t conv_bwd_workspace_bytes(const ConvGeom &g, int in_dtype, bool allow_split);
// cur [NB, Co, Hp, Wp] and the window choice (0..3) per pooled current
hipError_t launch_conv_pool_fwd(const ConvGeom &g, const void *x, int in_dtype, const void *w,
                                const float *bias, float *cur, uint8_t *arg, bool allow_split,
                                void *ws, size_t ws_bytes, hipStream_t s);
// grad_w [Co, Ci, 5, 5] and grad_x [NB, Ci, H, W] (either may be NULL)
hipError_t launch_conv_pool_bwd(const ConvGeom &g, const float *dI, const uint8_t *arg,
                                const void *x, int in_dtype, const void *w, bool allow_split,
                                float *grad_w, float *grad_x, void *ws, size_t ws_bytes,
                                hipStream_t s);

// ---- fused small-batch step (fused.hip) ---------------------------------------
constexpr int kFusedMaxNpw = 16;                 // hidden neurons per workgroup
constexpr size_t kFusedMaxLds = 160 * 1024 - 4096;  // dynamic LDS per workgroup
constexpr int kFusedMaxOut = 16;                 // readout neurons (one MFMA block)
struct FusedPlan {
    bool ok;
    int npw, grid;
    size_t lds, ws_bytes;
};
FusedPlan fused_plan(int T, int B, int n_in, int n_hid, int n_out);
struct FusedStep {
    int T, B, n_in, n_hid, n_out, P;
    int neuron0, neuron1;
    bool rs0, rs1;
    float alpha0, beta0, thr0, slope0, alpha1, beta1, thr1, slope1;
    int loss_kind;
    unsigned wait_limit;
    const uint8_t *x;
    const float *W0, *b0, *W1, *b1;
    const int32_t *labels;
    const float *targets;
    float *loss, *counts, *gW0, *gb0, *gW1, *gb1;
    uint8_t *spk;
    int32_t *status;
};
hipError_t launch_fused_step(const FusedStep &f, void *ws, hipStream_t s);

}  // namespace snn
