// Host side of the C ABI (include/snn.h): argument validation, workspace
// layout and the order of kernel launches for one layer.
#include <math.h>
#include <string.h>

#include "snn_internal.hpp"

using namespace snn;

namespace {

bool aligned16(const void *p) { return (((uintptr_t)p) & 15u) == 0; }

bool finite(float x) { return isfinite(x) != 0; }

int64_t rows(const snn_layer_desc *d) { return (int64_t)d->T * d->B; }

ConvGeom conv_geom(const snn_layer_desc *d) {
    ConvGeom g{};
    g.NB = (int)rows(d);
    g.Ci = d->c_in;
    g.H = d->h_in;
    g.W = d->w_in;
    g.Co = d->c_out;
    g.Ho = d->h_in - 4;
    g.Wo = d->w_in - 4;
    g.Hp = g.Ho / 2;
    g.Wp = g.Wo / 2;
    return g;
}

// Validates a layer descriptor; nothing here touches the device.
snn_status check_desc(const snn_layer_desc *d) {
    if (!d) return SNN_ERR_NULL;
    if (d->flags & ~SNN_FLAG_FP32_MFMA) return SNN_ERR_UNSUPPORTED;
    if (d->T < 0 || d->B < 0 || d->n_in < 0 || d->n_out < 0) return SNN_ERR_SHAPE;
    if (d->neuron != SNN_LEAKY && d->neuron != SNN_SYNAPTIC && d->neuron != SNN_RLEAKY)
        return SNN_ERR_UNSUPPORTED;
    if (d->reset_grad != SNN_RESET_DETACHED && d->reset_grad != SNN_RESET_SURROGATE)
        return SNN_ERR_UNSUPPORTED;
    if (!finite(d->beta) || !finite(d->alpha) || !finite(d->threshold) || !finite(d->slope) ||
        d->slope < 0.f)
        return SNN_ERR_SHAPE;
    if (d->out_dtype != SNN_U8 && d->out_dtype != SNN_F16 && d->out_dtype != SNN_SPK_BITS)
        return SNN_ERR_DTYPE;
    if (d->out_dtype == SNN_SPK_BITS && d->n_out % 64 != 0) return SNN_ERR_SHAPE;
    if (d->grad_dtype != SNN_F32 && d->grad_dtype != SNN_F16 && d->grad_dtype != SNN_BF16)
        return SNN_ERR_DTYPE;
    const int64_t TB = (int64_t)d->T * d->B;
    if (TB > INT32_MAX) return SNN_ERR_SHAPE;
    switch (d->synapse) {
        case SNN_SYN_DENSE:
            if (d->n_in < 1 || d->n_out < 1) return SNN_ERR_SHAPE;
            if (d->in_dtype != SNN_U8 && d->in_dtype != SNN_F32 && d->in_dtype != SNN_F16 &&
                !(d->in_dtype == SNN_BF16 && d->w_dtype == SNN_F32))
                return SNN_ERR_DTYPE;
            if (d->w_dtype != SNN_F32 && d->w_dtype != SNN_F16) return SNN_ERR_DTYPE;
            break;
        case SNN_SYN_CONV5_POOL2: {
            if (d->c_in < 1 || d->c_out < 1 || d->h_in < 6 || d->w_in < 6) return SNN_ERR_SHAPE;
            const int64_t hp = (d->h_in - 4) / 2, wp = (d->w_in - 4) / 2;
            if ((int64_t)d->c_in * d->h_in * d->w_in != d->n_in) return SNN_ERR_SHAPE;
            if ((int64_t)d->c_out * hp * wp != d->n_out) return SNN_ERR_SHAPE;
            if (d->in_dtype != SNN_U8 && d->in_dtype != SNN_F32) return SNN_ERR_DTYPE;
            if (d->w_dtype != SNN_F32 || d->grad_dtype != SNN_F32) return SNN_ERR_DTYPE;
            if (d->c_out > 2047) return SNN_ERR_UNSUPPORTED;
            if (!conv_fits_int32(conv_geom(d))) return SNN_ERR_SHAPE;
            break;
        }
        case SNN_SYN_NONE:
            if (d->n_in != d->n_out || d->n_out < 1) return SNN_ERR_SHAPE;
            if (d->in_dtype != SNN_F32) return SNN_ERR_DTYPE;
            if (d->grad_dtype != SNN_F32) return SNN_ERR_DTYPE;
            break;
        default:
            return SNN_ERR_UNSUPPORTED;
    }
    if (TB * (int64_t)(d->n_in > d->n_out ? d->n_in : d->n_out) > ((int64_t)1 << 40))
        return SNN_ERR_SHAPE;
    return SNN_OK;
}

// ---- saved state ------------------------------------------------------------
// [currents fp32 T*B*n_out (not for SYN_NONE, whose x holds them)]
// [checkpoints: planes (u; i too for SNN_SYNAPTIC) x count x B*n_out fp32]
// [pool selection u8 T*B*n_out (conv only)], each on a 256-byte boundary
snn_saved_layout saved_layout(const snn_layer_desc *d) {
    snn_saved_layout l{};
    const size_t el = (size_t)rows(d) * d->n_out;
    l.cur_bytes = d->synapse == SNN_SYN_NONE ? 0 : align_up(el * sizeof(float));
    l.ckpt_interval = kCheckpointInterval;
    l.ckpt_count = (int32_t)neuron_ckpt_count(d->T);
    l.ckpt_planes = d->neuron == SNN_SYNAPTIC ? 2 : 1;
    l.ckpt_offset = l.cur_offset + l.cur_bytes;
    l.ckpt_bytes = align_up((size_t)l.ckpt_planes * l.ckpt_count * d->B * d->n_out * sizeof(float));
    l.pool_offset = l.ckpt_offset + l.ckpt_bytes;
    l.pool_bytes = d->synapse == SNN_SYN_CONV5_POOL2 ? align_up(el) : 0;
    l.bytes = l.pool_offset + l.pool_bytes;
    return l;
}

// spike x fp32 contractions may use the exact three-pass bf16 kernels
bool split_ok(const snn_layer_desc *d) { return (d->flags & SNN_FLAG_FP32_MFMA) == 0; }

bool recurrent(const snn_layer_desc *d) { return d->neuron == SNN_RLEAKY; }

// ---- workspace layout ------------------------------------------------------
// forward:  [contraction workspace]
// backward: [dcur (grad_dtype) T*B*n_out][colsum fp32 B*n_out]
//           [dvcol fp32 B*n_out, recurrent neurons only][contraction workspace]
size_t fwd_ws(const snn_layer_desc *d) {
    if (d->synapse == SNN_SYN_CONV5_POOL2)
        return conv_fwd_workspace_bytes(conv_geom(d), d->in_dtype, split_ok(d));
    if (d->synapse != SNN_SYN_DENSE) return 0;
    return gemm_workspace_bytes((int)rows(d), d->n_out, d->n_in, d->in_dtype, d->w_dtype, true,
                                true, split_ok(d));
}
size_t dcur_bytes(const snn_layer_desc *d) {
    if (d->synapse == SNN_SYN_NONE) return 0;
    return align_up((size_t)rows(d) * d->n_out * dtype_bytes(d->grad_dtype));
}
size_t colsum_bytes(const snn_layer_desc *d) {
    return align_up((size_t)d->B * d->n_out * sizeof(float));
}
// An fp16 dL/dI is written scaled by a power of two S chosen per call from a
// bound of |dL/dI|: a device reduction over the upstream gradient (its
// partial maxima need grad_scale_workspace_bytes()) times the growth of the
// reverse recursion.
bool scaled_grad(const snn_layer_desc *d) { return d->grad_dtype == SNN_F16; }
size_t scale_scratch_bytes(const snn_layer_desc *d) {
    return scaled_grad(d) ? align_up(grad_scale_workspace_bytes()) : 0;
}
// |dL/dI_t| <= G * growth with G = max |g|: each step of the reverse
// recursion multiplies the carried adjoint by beta - r thr s, s in (0, 1]
// (|.| <= c = max(|beta|, |beta - r thr|)), and adds g s (|g s| <= G), so
// |lam_t| <= G sum_{k<T} c^k; the current-based neuron's lami sums lam with
// powers of alpha.  The recurrent neuron's carry depends on its weights v
// (device data): no fp16 gradient operand for it.
double grad_growth(const snn_layer_desc *d) {
    auto geo = [&](double q) {
        if (q == 1.0) return (double)d->T;
        return (1.0 - pow(q, (double)d->T)) / (1.0 - q);
    };
    const double r = d->reset_grad == SNN_RESET_SURROGATE ? 1.0 : 0.0;
    const double c = fmax(fabs((double)d->beta), fabs((double)d->beta - r * d->threshold));
    double F = geo(c);
    if (d->neuron == SNN_SYNAPTIC) F *= geo(fabs((double)d->alpha));
    return F;
}
bool scale_ok(const snn_layer_desc *d) {
    if (!scaled_grad(d)) return true;
    if (d->neuron == SNN_RLEAKY) return false;
    const double F = grad_growth(d);
    return isfinite(F) && F <= 1e30;
}
// per-column sums of the neuron backward: dL/dI (bias) and, for the recurrent
// neuron, lam_{t+1} z_t (recurrent weight); the partial maxima of an fp16
// dL/dI's scale
size_t neuron_ws(const snn_layer_desc *d) {
    return colsum_bytes(d) * (recurrent(d) ? 2 : 1) + scale_scratch_bytes(d);
}
// the device scalar S of an fp16 dL/dI inside the layer workspace
size_t scale_slot_bytes(const snn_layer_desc *d) { return scaled_grad(d) ? kAlign : 0; }
// Weight and input gradients of a dense layer.  Large contractions whose
// operands are stored M/N-contiguous (dI and x for dW, W for dx) are
// transposed once into the workspace so that they run K-contiguous on the
// 16-bit matrix cores; an fp32 dI is transposed straight into its three exact
// bf16 planes.
constexpr double kTransposeFlops = 1073741824.0;  // 2 M N K above which it pays

struct DwPlan {
    bool transposed;
    bool planes;       // fp32 dI as three bf16 planes in its own layout (asynchronous kernel)
    int a_dtype;       // dtype of the transposed dI operand
    size_t dit_bytes;  // dI^T (planes for fp32)
    size_t xt_bytes;   // x^T
    size_t gemm_bytes;
};

GemmArgs dw_probe_kc(const snn_layer_desc *d) {
    GemmArgs g{};
    g.M = d->n_out; g.N = d->n_in; g.K = (int)rows(d);
    g.a_dtype = d->grad_dtype == SNN_F32 ? kPlanes3 : d->grad_dtype; g.a_kc = true;
    g.b_dtype = d->in_dtype; g.b_kc = true;
    return g;
}

DwPlan dw_plan(const snn_layer_desc *d) {
    DwPlan p{};
    const int M = (int)rows(d);
    const GemmArgs kc = dw_probe_kc(d);
    // A layer with few outputs reads its operands in their own layouts, and
    // so does an fp32 dL/dI against spikes over at most 8192 rows: the 16-bit
    // kernel stages both M/N-contiguous tiles in LDS as they are and reads
    // transposed fragments (measured: 42 against 34 + 17 us of contraction and
    // transposes at 3200 rows, 127 against 85 + 34 us at 12800 rows).
    const bool mn_direct = d->grad_dtype == SNN_F32 && d->in_dtype == SNN_U8 && M <= 8192;
    // A 16-bit dL/dI against 16-bit or spike x on the asynchronous pipeline:
    // the tiles are staged M/N-contiguous as they are and read with
    // transposing LDS loads, so no operand is transposed in global memory.
    GemmArgs mn{};
    mn.M = d->n_out; mn.N = d->n_in; mn.K = M;
    mn.a_dtype = d->grad_dtype; mn.a_kc = false; mn.lda = d->n_out;
    mn.b_dtype = d->in_dtype; mn.b_kc = false; mn.ldb = d->n_in;
    mn.allow_split = split_ok(d);
    const bool async_mn = gemm_async_applies(mn);
    p.planes = async_mn && d->grad_dtype == SNN_F32;
    p.transposed = split_ok(d) && gemm16_applies(kc) && d->n_out > 16 && !mn_direct && !async_mn &&
                   2.0 * M * d->n_in * d->n_out >= kTransposeFlops;
    if (p.transposed) {
        p.a_dtype = kc.a_dtype;
        p.dit_bytes = align_up((size_t)M * d->n_out * dtype_bytes(kc.a_dtype));
        p.xt_bytes = align_up((size_t)M * d->n_in * dtype_bytes(d->in_dtype));
        p.gemm_bytes = gemm_workspace_bytes(kc.M, kc.N, kc.K, kc.a_dtype, kc.b_dtype, true, true, true);
    } else {
        p.gemm_bytes = gemm_workspace_bytes(d->n_out, d->n_in, M, d->grad_dtype, d->in_dtype,
                                            false, false, split_ok(d));
    }
    return p;
}

// bytes of the weight gradient's dL/dI operand as the reverse scan can write
// it: transposed ([planes][n_out][T*B] 16-bit) or, for an fp32 dL/dI read in
// its own layout, its three bf16 planes [3][T*B][n_out]; 0 when the layer's
// weight gradient contracts neither
size_t dcur_t_bytes(const snn_layer_desc *d) {
    if (d->synapse != SNN_SYN_DENSE || rows(d) == 0) return 0;
    const DwPlan p = dw_plan(d);
    if (p.planes) return align_up((size_t)3 * rows(d) * d->n_out * sizeof(uint16_t));
    return p.transposed ? p.dit_bytes : 0;
}
bool dcur_t_planes(const snn_layer_desc *d) {
    return d->synapse == SNN_SYN_DENSE && rows(d) > 0 && dw_plan(d).planes;
}
// the layer call has the reverse scan write the planes (in its workspace)
size_t layer_planes_bytes(const snn_layer_desc *d) { return dcur_t_planes(d) ? dcur_t_bytes(d) : 0; }

struct DxPlan {
    bool transposed;
    size_t wt_bytes;  // W^T
    size_t gemm_bytes;
};

DxPlan dx_plan(const snn_layer_desc *d) {
    DxPlan p{};
    const int M = (int)rows(d);
    GemmArgs kc{};
    kc.M = M; kc.N = d->n_in; kc.K = d->n_out;
    kc.a_dtype = d->grad_dtype; kc.a_kc = true;
    kc.b_dtype = d->w_dtype; kc.b_kc = true;
    // a layer with few outputs (short contraction) reads W in its own layout
    p.transposed = split_ok(d) && gemm16_applies(kc) && d->n_out > 16 &&
                   2.0 * M * d->n_in * d->n_out >= kTransposeFlops;
    if (p.transposed) {
        p.wt_bytes = align_up((size_t)d->n_in * d->n_out * dtype_bytes(d->w_dtype));
        p.gemm_bytes = gemm_workspace_bytes(M, d->n_in, d->n_out, d->grad_dtype, d->w_dtype, true,
                                            true, true);
    } else {
        p.gemm_bytes = gemm_workspace_bytes(M, d->n_in, d->n_out, d->grad_dtype, d->w_dtype, true,
                                            false, split_ok(d));
    }
    return p;
}

size_t bwd_gemm_ws(const snn_layer_desc *d) {
    if (d->synapse == SNN_SYN_CONV5_POOL2)
        return conv_bwd_workspace_bytes(conv_geom(d), d->in_dtype, split_ok(d));
    if (d->synapse != SNN_SYN_DENSE) return 0;
    const DwPlan w = dw_plan(d);
    const DxPlan x = dx_plan(d);
    const size_t dw = w.dit_bytes + w.xt_bytes + w.gemm_bytes;
    const size_t dx = x.wt_bytes + x.gemm_bytes;
    return dw > dx ? dw : dx;
}
size_t bwd_ws(const snn_layer_desc *d) {
    return dcur_bytes(d) + neuron_ws(d) + scale_slot_bytes(d) + layer_planes_bytes(d) +
           bwd_gemm_ws(d);
}

snn_status hip_status(hipError_t e) { return e == hipSuccess ? SNN_OK : SNN_ERR_HIP; }

snn_status check_grad(const snn_layer_desc *d, const snn_grad_in *g) {
    if (!g) return SNN_ERR_NULL;
    if (g->kind == SNN_GRAD_FULL || g->kind == SNN_GRAD_BCAST) {
        if (!g->g) return SNN_ERR_NULL;
        if (g->n_up != 0) return SNN_ERR_UNSUPPORTED;
        if (!aligned16(g->g)) return SNN_ERR_ALIGN;
        return SNN_OK;
    }
    if (g->kind != SNN_GRAD_FOLD) return SNN_ERR_UNSUPPORTED;
    if (!g->dcur_up || !g->w_up) return SNN_ERR_NULL;
    if (g->n_up < 1 || g->n_up > 16) return SNN_ERR_SHAPE;
    if (g->dcur_up_dtype != SNN_F32 && g->dcur_up_dtype != SNN_BF16 && g->dcur_up_dtype != SNN_F16)
        return SNN_ERR_DTYPE;
    if (g->w_up_dtype != SNN_F32 && g->w_up_dtype != SNN_F16) return SNN_ERR_DTYPE;
    if (!aligned16(g->dcur_up) || !aligned16(g->w_up)) return SNN_ERR_ALIGN;
    if (!neuron_fold_supported(d->n_out)) return SNN_ERR_UNSUPPORTED;
    return SNN_OK;
}

snn_status check_loss(int32_t kind, int32_t B, int32_t K, int32_t P, const float *counts,
                      const int32_t *labels, const float *targets, const float *loss,
                      const float *grad_counts) {
    if (kind != SNN_LOSS_CE_COUNT && kind != SNN_LOSS_MSE_COUNT) return SNN_ERR_UNSUPPORTED;
    if (B < 1 || K < 1 || P < 1 || (int64_t)K * P > INT32_MAX) return SNN_ERR_SHAPE;
    if (!counts || !loss) return SNN_ERR_NULL;
    if (kind == SNN_LOSS_CE_COUNT && !labels) return SNN_ERR_NULL;
    if (kind == SNN_LOSS_MSE_COUNT && !targets) return SNN_ERR_NULL;
    if (!aligned16(counts) || !aligned16(loss) || (labels && !aligned16(labels)) ||
        (targets && !aligned16(targets)) || (grad_counts && !aligned16(grad_counts)))
        return SNN_ERR_ALIGN;
    return SNN_OK;
}

BwdGrad bwd_grad(const snn_grad_in *g) {
    BwdGrad b{};
    b.mode = g->kind;
    b.g = g->kind == SNN_GRAD_FOLD ? nullptr : g->g;
    if (g->kind == SNN_GRAD_FOLD) {
        b.dup = g->dcur_up;
        b.wup = g->w_up;
        b.nup = g->n_up;
        b.dt_up = g->dcur_up_dtype;
        b.dt_w = g->w_up_dtype;
    }
    return b;
}

}  // namespace

namespace {
snn_status check_fused(const snn_fused_desc *f, FusedPlan *plan) {
    if (!f) return SNN_ERR_NULL;
    const snn_layer_desc &h = f->hidden, &r = f->readout;
    snn_status st = check_desc(&h);
    if (st != SNN_OK) return st;
    st = check_desc(&r);
    if (st != SNN_OK) return st;
    if (h.synapse != SNN_SYN_DENSE || r.synapse != SNN_SYN_DENSE) return SNN_ERR_UNSUPPORTED;
    if (h.in_dtype != SNN_U8 || r.in_dtype != SNN_U8 || h.w_dtype != SNN_F32 ||
        r.w_dtype != SNN_F32 || h.out_dtype == SNN_SPK_BITS)
        return SNN_ERR_DTYPE;
    auto plain = [](int n) { return n == SNN_LEAKY || n == SNN_SYNAPTIC; };
    if (!plain(h.neuron) || !plain(r.neuron)) return SNN_ERR_UNSUPPORTED;
    if (r.n_in != h.n_out || r.T != h.T || r.B != h.B || h.T < 1 || h.B < 1)
        return SNN_ERR_SHAPE;
    if (f->loss_kind != SNN_LOSS_CE_COUNT && f->loss_kind != SNN_LOSS_MSE_COUNT)
        return SNN_ERR_UNSUPPORTED;
    if (f->pop < 1 || r.n_out % f->pop != 0 || f->reserved != 0) return SNN_ERR_SHAPE;
    if (r.n_out > kFusedMaxOut) return SNN_ERR_UNSUPPORTED;
    const FusedPlan p = fused_plan(h.T, h.B, h.n_in, h.n_out, r.n_out);
    if (!p.ok) return SNN_ERR_UNSUPPORTED;
    if (plan) *plan = p;
    return SNN_OK;
}
}  // namespace

extern "C" {

int snn_abi_version(void) { return SNN_ABI_VERSION; }

const char *snn_status_str(snn_status s) {
    switch (s) {
        case SNN_OK: return "ok";
        case SNN_ERR_NULL: return "required pointer is NULL";
        case SNN_ERR_SHAPE: return "invalid or inconsistent sizes";
        case SNN_ERR_DTYPE: return "unsupported dtype combination";
        case SNN_ERR_ALIGN: return "device pointer not 16-byte aligned";
        case SNN_ERR_UNSUPPORTED: return "not supported by this library";
        case SNN_ERR_WORKSPACE: return "workspace too small";
        case SNN_ERR_HIP: return "HIP launch failed";
    }
    return "unknown status";
}

size_t snn_layer_saved_bytes(const snn_layer_desc *d) {
    if (check_desc(d) != SNN_OK) return 0;
    return saved_layout(d).bytes;
}

size_t snn_layer_dcur_t_bytes(const snn_layer_desc *d) {
    if (check_desc(d) != SNN_OK) return 0;
    return dcur_t_bytes(d);
}

int32_t snn_layer_dcur_t_layout(const snn_layer_desc *d) {
    if (check_desc(d) != SNN_OK) return -1;
    return dcur_t_planes(d) ? SNN_DCUR_T_PLANES : SNN_DCUR_T_TRANSPOSED;
}

snn_status snn_layer_saved_layout(const snn_layer_desc *d, snn_saved_layout *out) {
    if (!out) return SNN_ERR_NULL;
    snn_status st = check_desc(d);
    if (st != SNN_OK) return st;
    *out = saved_layout(d);
    return SNN_OK;
}

size_t snn_layer_workspace_bytes(const snn_layer_desc *d) {
    if (check_desc(d) != SNN_OK) return 0;
    const size_t f = fwd_ws(d), b = bwd_ws(d);
    return f > b ? f : b;
}

snn_status snn_synapse_fwd(const snn_layer_desc *d, const void *x, const void *w,
                           const float *bias, float *cur, uint8_t *pool_arg, void *ws,
                           size_t ws_bytes, hipStream_t stream) {
    snn_status st = check_desc(d);
    if (st != SNN_OK) return st;
    if (d->synapse == SNN_SYN_NONE) return SNN_ERR_UNSUPPORTED;  // nothing to contract
    if (!x || !w || !cur) return SNN_ERR_NULL;
    if (!aligned16(x) || !aligned16(w) || !aligned16(cur) || (bias && !aligned16(bias)))
        return SNN_ERR_ALIGN;
    if (fwd_ws(d) > ws_bytes || (fwd_ws(d) > 0 && !ws)) return SNN_ERR_WORKSPACE;
    if (d->synapse == SNN_SYN_CONV5_POOL2 && !pool_arg) return SNN_ERR_NULL;
    if (rows(d) == 0) return SNN_OK;
    (void)hipGetLastError();
    if (d->synapse == SNN_SYN_CONV5_POOL2)
        return hip_status(launch_conv_pool_fwd(conv_geom(d), x, d->in_dtype, w, bias, cur,
                                               pool_arg, split_ok(d), ws, ws_bytes, stream));
    GemmArgs g{};
    g.M = (int)rows(d);
    g.N = d->n_out;
    g.K = d->n_in;
    g.A = x; g.lda = d->n_in; g.a_dtype = d->in_dtype; g.a_kc = true;
    g.B = w; g.ldb = d->n_in; g.b_dtype = d->w_dtype; g.b_kc = true;
    g.C = cur; g.ldc = d->n_out; g.bias = bias; g.allow_split = split_ok(d);
    return hip_status(launch_gemm(g, ws, ws_bytes, stream));
}

snn_status snn_neuron_fwd(const snn_layer_desc *d, const float *cur, const float *v,
                          void *spk_out, float *ckpt, float *u_out, float *counts,
                          hipStream_t stream) {
    snn_status st = check_desc(d);
    if (st != SNN_OK) return st;
    if (!cur || !spk_out) return SNN_ERR_NULL;
    if (neuron_ckpt_count(d->T) > 0 && d->B > 0 && !ckpt) return SNN_ERR_NULL;
    if (recurrent(d) && !v) return SNN_ERR_NULL;
    if (!recurrent(d)) v = nullptr;
    if (!aligned16(cur) || !aligned16(spk_out) || (ckpt && !aligned16(ckpt)) ||
        (u_out && !aligned16(u_out)) || (counts && !aligned16(counts)) || (v && !aligned16(v)))
        return SNN_ERR_ALIGN;
    (void)hipGetLastError();
    if (rows(d) == 0) {
        // counts over zero time steps are 0
        if (counts) return hip_status(launch_fill_zero(counts, (int64_t)d->B * d->n_out, stream));
        return SNN_OK;
    }
    const int64_t C = (int64_t)d->B * d->n_out;
    return hip_status(launch_neuron_fwd(d->neuron, d->T, C, d->n_out, d->alpha, d->beta,
                                        d->threshold, v, cur, spk_out, d->out_dtype, u_out, ckpt,
                                        counts, stream));
}

snn_status snn_neuron_bwd(const snn_layer_desc *d, const snn_grad_in *grad, const float *v,
                          const float *cur, const float *ckpt, void *dcur, void *dcur_t,
                          float *dcur_scale, float *grad_b, float *grad_v, void *ws,
                          size_t ws_bytes, hipStream_t stream) {
    snn_status st = check_desc(d);
    if (st != SNN_OK) return st;
    if ((st = check_grad(d, grad)) != SNN_OK) return st;
    if (!cur || (!dcur && !dcur_t)) return SNN_ERR_NULL;
    if (dcur_t && (d->synapse != SNN_SYN_DENSE || !aligned16(dcur_t)))
        return d->synapse != SNN_SYN_DENSE ? SNN_ERR_UNSUPPORTED : SNN_ERR_ALIGN;
    if (neuron_ckpt_count(d->T) > 0 && d->B > 0 && !ckpt) return SNN_ERR_NULL;
    if (ckpt && !aligned16(ckpt)) return SNN_ERR_ALIGN;
    if (scaled_grad(d)) {
        if (!dcur_scale) return SNN_ERR_NULL;
        if (!aligned16(dcur_scale)) return SNN_ERR_ALIGN;
        if (!scale_ok(d)) return SNN_ERR_UNSUPPORTED;
    } else {
        dcur_scale = nullptr;
    }
    if (recurrent(d) && !v) return SNN_ERR_NULL;
    if (!recurrent(d)) {
        if (grad_v) return SNN_ERR_SHAPE;  // no recurrent weight to differentiate
        v = nullptr;
    }
    if (!aligned16(cur) || (dcur && !aligned16(dcur)) || (grad_b && !aligned16(grad_b)) ||
        (v && !aligned16(v)) || (grad_v && !aligned16(grad_v)))
        return SNN_ERR_ALIGN;
    if (grad_b && d->synapse == SNN_SYN_NONE) return SNN_ERR_SHAPE;  // no bias to differentiate
    const size_t sums = (grad_b ? colsum_bytes(d) : 0) + (grad_v ? colsum_bytes(d) : 0);
    const size_t need = sums + scale_scratch_bytes(d);
    if (need > ws_bytes || (need > 0 && !ws)) return SNN_ERR_WORKSPACE;
    (void)hipGetLastError();
    if (rows(d) == 0) {
        hipError_t e = hipSuccess;
        if (grad_b) {
            const int64_t nb = d->synapse == SNN_SYN_CONV5_POOL2 ? d->c_out : d->n_out;
            e = launch_fill_zero(grad_b, nb, stream);
        }
        if (grad_v && e == hipSuccess) e = launch_fill_zero(grad_v, d->n_out, stream);
        // an empty gradient: its scale is 1
        if (dcur_scale && e == hipSuccess)
            e = launch_grad_scale(d->T, (int64_t)d->B * d->n_out, bwd_grad(grad), d->B, 1.0,
                                  dcur_scale, reinterpret_cast<float *>(
                                      reinterpret_cast<char *>(ws) +
                                      (grad_b ? colsum_bytes(d) : 0) + (grad_v ? colsum_bytes(d) : 0)),
                                  stream);
        return hip_status(e);
    }
    const int64_t C = (int64_t)d->B * d->n_out;
    char *wsb = reinterpret_cast<char *>(ws);
    float *colsum = grad_b ? reinterpret_cast<float *>(wsb) : nullptr;
    float *dvcol = grad_v ? reinterpret_cast<float *>(wsb + (grad_b ? colsum_bytes(d) : 0))
                          : nullptr;
    const BwdGrad bg = bwd_grad(grad);
    hipError_t e = hipSuccess;
    if (dcur_scale) {
        e = launch_grad_scale(d->T, C, bg, d->B, grad_growth(d), dcur_scale,
                              reinterpret_cast<float *>(wsb + sums), stream);
        if (e != hipSuccess) return SNN_ERR_HIP;
    }
    e = launch_neuron_bwd(d->neuron, d->reset_grad, d->T, C, d->n_out, d->alpha, d->beta,
                          d->threshold, d->slope, v, cur, ckpt, bg, d->B, dcur, dcur_t,
                          dcur_t_planes(d), d->grad_dtype, dcur_scale, colsum, dvcol, stream);
    if (e != hipSuccess) return SNN_ERR_HIP;
    if (grad_b) {
        int F = d->n_out, P = 1;
        if (d->synapse == SNN_SYN_CONV5_POOL2) {
            F = d->c_out;
            P = d->n_out / d->c_out;
        }
        e = launch_bias_reduce(d->B, F, P, colsum, grad_b, stream);
        if (e != hipSuccess) return SNN_ERR_HIP;
    }
    // dL/dv[n] = sum over the batch of the per-column sums, fixed order
    if (grad_v) e = launch_bias_reduce(d->B, d->n_out, 1, dvcol, grad_v, stream);
    return hip_status(e);
}

snn_status snn_synapse_bwd(const snn_layer_desc *d, const void *dcur, const void *dcur_t,
                           const float *dcur_scale, const uint8_t *pool_arg, const void *x,
                           const void *w, float *grad_w, float *grad_x, void *ws,
                           size_t ws_bytes, hipStream_t stream) {
    snn_status st = check_desc(d);
    if (st != SNN_OK) return st;
    if (d->synapse == SNN_SYN_NONE) return SNN_ERR_UNSUPPORTED;
    // dcur_t (the transposed weight-gradient operand) serves the weight
    // gradient when the layer's plan contracts it; dcur everything else
    const bool use_t = dcur_t && grad_w && dcur_t_bytes(d) > 0;
    if (dcur_t && !aligned16(dcur_t)) return SNN_ERR_ALIGN;
    if (!dcur && (grad_x || (grad_w && !use_t))) return SNN_ERR_NULL;
    if (!dcur && !dcur_t) return SNN_ERR_NULL;
    if (scaled_grad(d)) {
        if (!dcur_scale) return SNN_ERR_NULL;
        if (!aligned16(dcur_scale)) return SNN_ERR_ALIGN;
    } else {
        dcur_scale = nullptr;
    }
    if ((grad_w && !x) || (grad_x && !w)) return SNN_ERR_NULL;
    if ((dcur && !aligned16(dcur)) || (x && !aligned16(x)) || (w && !aligned16(w)) ||
        (grad_w && !aligned16(grad_w)) || (grad_x && !aligned16(grad_x)))
        return SNN_ERR_ALIGN;
    const size_t need = bwd_gemm_ws(d);
    if (need > ws_bytes || (need > 0 && !ws)) return SNN_ERR_WORKSPACE;
    if (d->synapse == SNN_SYN_CONV5_POOL2 && !pool_arg) return SNN_ERR_NULL;
    if (rows(d) == 0) {
        // empty batch: the weight gradient is an empty sum
        if (grad_w)
            return hip_status(launch_fill_zero(grad_w, (int64_t)d->n_out * d->n_in, stream));
        return SNN_OK;
    }
    (void)hipGetLastError();
    if (d->synapse == SNN_SYN_CONV5_POOL2)
        return hip_status(launch_conv_pool_bwd(conv_geom(d), reinterpret_cast<const float *>(dcur),
                                               pool_arg, x, d->in_dtype, w, split_ok(d), grad_w,
                                               grad_x, ws, ws_bytes, stream));
    const int M = (int)rows(d);
    char *wsb = reinterpret_cast<char *>(ws);
    if (grad_w) {
        // dW[o,i] = sum_m dI[m,o] x[m,i], K = T*B
        const DwPlan pl = dw_plan(d);
        GemmArgs g{};
        g.M = d->n_out; g.N = d->n_in; g.K = M;
        g.C = grad_w; g.ldc = d->n_in; g.bias = nullptr; g.allow_split = split_ok(d);
        g.c_div = dcur_scale;
        hipError_t e;
        if (pl.transposed) {
            // K = T*B in the order k = b*T + t on both operands: the order in
            // which the reverse scan writes dL/dI transposed (one lane's
            // column is one row there)
            char *dit = wsb, *xt = wsb + pl.dit_bytes;
            const bool planes = pl.a_dtype == kPlanes3;
            const void *A = dcur_t;
            if (!use_t) {
                e = launch_transpose(M, d->n_out, dcur, d->n_out, (int)dtype_bytes(d->grad_dtype),
                                     dit, M, planes, (int64_t)M * d->n_out, stream, d->T);
                if (e != hipSuccess) return SNN_ERR_HIP;
                A = dit;
            }
            e = launch_transpose(M, d->n_in, x, d->n_in, (int)dtype_bytes(d->in_dtype), xt, M, false,
                                 0, stream, d->T);
            if (e != hipSuccess) return SNN_ERR_HIP;
            g.A = A; g.lda = M; g.a_dtype = pl.a_dtype; g.a_kc = true;
            g.a_ps = (int64_t)M * d->n_out;
            g.B = xt; g.ldb = M; g.b_dtype = d->in_dtype; g.b_kc = true;
            e = launch_gemm(g, xt + pl.xt_bytes, ws_bytes - pl.dit_bytes - pl.xt_bytes, stream);
        } else {
            // both operands stored with the output index contiguous; an fp32
            // dI as the three bf16 planes the reverse scan wrote, else split
            // into planes in the workspace
            g.A = dcur; g.lda = d->n_out; g.a_dtype = d->grad_dtype; g.a_kc = false;
            if (use_t && pl.planes) {
                g.A = dcur_t;
                g.a_dtype = kPlanes3;
                g.a_ps = (int64_t)M * d->n_out;
            }
            g.B = x; g.ldb = d->n_in; g.b_dtype = d->in_dtype; g.b_kc = false;
            e = launch_gemm(g, ws, ws_bytes, stream);
        }
        if (e != hipSuccess) return SNN_ERR_HIP;
    }
    if (grad_x) {
        // dx[m,i] = sum_o dI[m,o] W[o,i]
        const DxPlan pl = dx_plan(d);
        GemmArgs g{};
        g.M = M; g.N = d->n_in; g.K = d->n_out;
        g.A = dcur; g.lda = d->n_out; g.a_dtype = d->grad_dtype; g.a_kc = true;
        g.C = grad_x; g.ldc = d->n_in; g.bias = nullptr; g.allow_split = split_ok(d);
        g.c_div = dcur_scale;
        hipError_t e;
        if (pl.transposed) {
            e = launch_transpose(d->n_out, d->n_in, w, d->n_in, (int)dtype_bytes(d->w_dtype), wsb,
                                 d->n_out, false, 0, stream);
            if (e != hipSuccess) return SNN_ERR_HIP;
            g.B = wsb; g.ldb = d->n_out; g.b_dtype = d->w_dtype; g.b_kc = true;
            e = launch_gemm(g, wsb + pl.wt_bytes, ws_bytes - pl.wt_bytes, stream);
        } else {
            g.B = w; g.ldb = d->n_in; g.b_dtype = d->w_dtype; g.b_kc = false;
            e = launch_gemm(g, ws, ws_bytes, stream);
        }
        if (e != hipSuccess) return SNN_ERR_HIP;
    }
    return SNN_OK;
}

snn_status snn_layer_fwd(const snn_layer_desc *d, const void *x, const void *w,
                         const float *bias, const float *v, void *spk_out, void *saved,
                         float *counts, void *ws, size_t ws_bytes, hipStream_t stream) {
    snn_status st = check_desc(d);
    if (st != SNN_OK) return st;
    if (!x || !spk_out || !saved) return SNN_ERR_NULL;
    if (d->synapse != SNN_SYN_NONE && !w) return SNN_ERR_NULL;
    if (recurrent(d) && !v) return SNN_ERR_NULL;
    if (v && recurrent(d) && !aligned16(v)) return SNN_ERR_ALIGN;
    if (!aligned16(x) || !aligned16(spk_out) || !aligned16(saved) || (w && !aligned16(w)) ||
        (bias && !aligned16(bias)) || (counts && !aligned16(counts)))
        return SNN_ERR_ALIGN;
    if (fwd_ws(d) > ws_bytes) return SNN_ERR_WORKSPACE;
    const snn_saved_layout l = saved_layout(d);
    char *sb = reinterpret_cast<char *>(saved);
    float *ckpt = reinterpret_cast<float *>(sb + l.ckpt_offset);
    if (d->synapse == SNN_SYN_NONE)
        return snn_neuron_fwd(d, reinterpret_cast<const float *>(x), v, spk_out, ckpt, nullptr,
                              counts, stream);
    float *cur = reinterpret_cast<float *>(sb + l.cur_offset);
    uint8_t *arg = nullptr;
    if (d->synapse == SNN_SYN_CONV5_POOL2) arg = reinterpret_cast<uint8_t *>(sb + l.pool_offset);
    st = snn_synapse_fwd(d, x, w, bias, cur, arg, ws, ws_bytes, stream);
    if (st != SNN_OK) return st;
    return snn_neuron_fwd(d, cur, v, spk_out, ckpt, nullptr, counts, stream);
}

snn_status snn_layer_bwd(const snn_layer_desc *d, const snn_grad_in *grad, const void *x,
                         const void *w, const float *v, const void *saved, float *grad_w,
                         float *grad_b, float *grad_v, float *grad_x, void *ws,
                         size_t ws_bytes, hipStream_t stream) {
    snn_status st = check_desc(d);
    if (st != SNN_OK) return st;
    if ((st = check_grad(d, grad)) != SNN_OK) return st;
    if (!saved) return SNN_ERR_NULL;
    if (!aligned16(saved)) return SNN_ERR_ALIGN;
    const snn_saved_layout l = saved_layout(d);
    const char *sb = reinterpret_cast<const char *>(saved);
    const float *ckpt = reinterpret_cast<const float *>(sb + l.ckpt_offset);
    if (d->synapse == SNN_SYN_NONE) {
        if (grad_w || grad_b) return SNN_ERR_SHAPE;
        if (!grad_x || !x) return SNN_ERR_NULL;
        // the currents are the layer's input
        return snn_neuron_bwd(d, grad, v, reinterpret_cast<const float *>(x), ckpt, grad_x,
                              nullptr, nullptr, nullptr, grad_v, ws, ws_bytes, stream);
    }
    const float *cur = reinterpret_cast<const float *>(sb + l.cur_offset);
    if (grad_w && !x) return SNN_ERR_NULL;
    if (grad_x && !w) return SNN_ERR_NULL;
    if (bwd_ws(d) > ws_bytes || !ws) return SNN_ERR_WORKSPACE;
    char *base = reinterpret_cast<char *>(ws);
    void *dcur = base;
    char *colsum = base + dcur_bytes(d);
    float *scale = scaled_grad(d) ? reinterpret_cast<float *>(colsum + neuron_ws(d)) : nullptr;
    char *planes = colsum + neuron_ws(d) + scale_slot_bytes(d);
    char *gws = planes + layer_planes_bytes(d);
    // Where the weight gradient takes a transposed operand (fp32 dL/dI as
    // three bf16 parts), the reverse scan could write it itself (dcur_t), but
    // its rows are written in runs of one chunk (16 steps, 32 bytes) per
    // lane, which measured slower than the row-major write plus one
    // transpose, so the layer call keeps the transpose.  Where it takes an
    // fp32 dL/dI in its own layout, the scan writes the three bf16 planes
    // (coalesced like dL/dI itself) instead of the fp32 values, which only
    // the input gradient still needs.
    void *dcur_t = nullptr;
    void *dcur_rm = dcur;
    if (grad_w && layer_planes_bytes(d) > 0) {
        dcur_t = planes;
        if (!grad_x) dcur_rm = nullptr;
    }
    st = snn_neuron_bwd(d, grad, v, cur, ckpt, dcur_rm, dcur_t, scale, grad_b, grad_v, colsum,
                        neuron_ws(d), stream);
    if (st != SNN_OK) return st;
    if (!grad_w && !grad_x) return SNN_OK;
    const uint8_t *arg = nullptr;
    if (d->synapse == SNN_SYN_CONV5_POOL2) arg = reinterpret_cast<const uint8_t *>(sb + l.pool_offset);
    return snn_synapse_bwd(d, dcur_rm, dcur_t, scale, arg, x, w, grad_w, grad_x, gws,
                           bwd_gemm_ws(d), stream);
}

size_t snn_loss_workspace_bytes(int32_t kind, int32_t B, int32_t K) {
    if (kind != SNN_LOSS_CE_COUNT && kind != SNN_LOSS_MSE_COUNT) return 0;
    return loss_workspace_bytes(kind, B, K);
}

snn_status snn_loss(int32_t kind, int32_t B, int32_t K, int32_t P, const float *counts,
                    const int32_t *labels, const float *targets, float *loss,
                    float *grad_counts, void *ws, size_t ws_bytes, hipStream_t stream) {
    snn_status st = check_loss(kind, B, K, P, counts, labels, targets, loss, grad_counts);
    if (st != SNN_OK) return st;
    const size_t need = loss_workspace_bytes(kind, B, K);
    if (need > ws_bytes || (need > 0 && !ws)) return SNN_ERR_WORKSPACE;
    (void)hipGetLastError();
    return hip_status(launch_loss(kind, B, K, P, counts, labels, targets, loss, grad_counts, ws,
                                  stream));
}

snn_status snn_loss_noalloc(int32_t kind, int32_t B, int32_t K, int32_t P, const float *counts,
                            const int32_t *labels, const float *targets, float *loss,
                            float *grad_counts, hipStream_t stream) {
    snn_status st = check_loss(kind, B, K, P, counts, labels, targets, loss, grad_counts);
    if (st != SNN_OK) return st;
    if (loss_workspace_bytes(kind, B, K) > kLossScratchBytes) return SNN_ERR_WORKSPACE;
    void *scratch = nullptr;
    if (loss_static_scratch(&scratch) != hipSuccess) return SNN_ERR_HIP;
    (void)hipGetLastError();
    return hip_status(launch_loss(kind, B, K, P, counts, labels, targets, loss, grad_counts,
                                  scratch, stream));
}


snn_status snn_fused_step_check(const snn_fused_desc *d) { return check_fused(d, nullptr); }

size_t snn_fused_step_workspace_bytes(const snn_fused_desc *d) {
    FusedPlan p{};
    return check_fused(d, &p) == SNN_OK ? p.ws_bytes : 0;
}

snn_status snn_fused_step(const snn_fused_desc *d, const uint8_t *x, const float *w0,
                          const float *b0, const float *w1, const float *b1,
                          const int32_t *labels, const float *targets, float *loss,
                          float *counts, uint8_t *spk_hidden, float *grad_w0, float *grad_b0,
                          float *grad_w1, float *grad_b1, int32_t *status, void *ws,
                          size_t ws_bytes, hipStream_t stream) {
    FusedPlan p{};
    snn_status st = check_fused(d, &p);
    if (st != SNN_OK) return st;
    if (!x || !w0 || !w1 || !status) return SNN_ERR_NULL;
    if (d->loss_kind == SNN_LOSS_CE_COUNT && !labels) return SNN_ERR_NULL;
    if (d->loss_kind == SNN_LOSS_MSE_COUNT && !targets) return SNN_ERR_NULL;
    for (const void *q : {(const void *)x, (const void *)w0, (const void *)b0, (const void *)w1,
                          (const void *)b1, (const void *)labels, (const void *)targets,
                          (const void *)loss, (const void *)counts, (const void *)spk_hidden,
                          (const void *)grad_w0,
                          (const void *)grad_b0, (const void *)grad_w1, (const void *)grad_b1,
                          (const void *)status, (const void *)ws})
        if (q && !aligned16(q)) return SNN_ERR_ALIGN;
    if (!ws || ws_bytes < p.ws_bytes) return SNN_ERR_WORKSPACE;
    const snn_layer_desc &h = d->hidden, &r = d->readout;
    FusedStep f{};
    f.T = h.T; f.B = h.B; f.n_in = h.n_in; f.n_hid = h.n_out; f.n_out = r.n_out; f.P = d->pop;
    f.neuron0 = h.neuron; f.neuron1 = r.neuron;
    f.rs0 = h.reset_grad == SNN_RESET_SURROGATE; f.rs1 = r.reset_grad == SNN_RESET_SURROGATE;
    f.alpha0 = h.alpha; f.beta0 = h.beta; f.thr0 = h.threshold; f.slope0 = h.slope;
    f.alpha1 = r.alpha; f.beta1 = r.beta; f.thr1 = r.threshold; f.slope1 = r.slope;
    f.loss_kind = d->loss_kind;
    f.wait_limit = d->wait_limit;
    f.x = x; f.W0 = w0; f.b0 = b0; f.W1 = w1; f.b1 = b1;
    f.labels = labels; f.targets = targets;
    f.loss = loss; f.counts = counts; f.spk = spk_hidden;
    f.gW0 = grad_w0; f.gb0 = grad_b0; f.gW1 = grad_w1; f.gb1 = grad_b1;
    f.status = status;
    (void)hipGetLastError();
    return hip_status(launch_fused_step(f, ws, stream));
}

snn_status snn_adamw(const snn_adamw_tensor *tensors, int32_t count,
                     const snn_adamw_hparams *hp, hipStream_t stream) {
    if (count < 0) return SNN_ERR_SHAPE;
    if (!hp || (count > 0 && !tensors)) return SNN_ERR_NULL;
    if (!finite(hp->lr) || !finite(hp->beta1) || !finite(hp->beta2) || !finite(hp->eps) ||
        !finite(hp->weight_decay) || hp->lr < 0.f || hp->beta1 < 0.f || hp->beta1 >= 1.f ||
        hp->beta2 < 0.f || hp->beta2 >= 1.f || hp->eps < 0.f || hp->weight_decay < 0.f ||
        hp->step < 1)
        return SNN_ERR_SHAPE;
    bool any = false;
    for (int i = 0; i < count; ++i) {
        const snn_adamw_tensor &t = tensors[i];
        if (t.n < 0 || t.n > ((int64_t)1 << 36)) return SNN_ERR_SHAPE;
        if (t.n == 0) continue;
        any = true;
        if (!t.param || !t.grad || !t.m || !t.v) return SNN_ERR_NULL;
        if (!aligned16(t.param) || !aligned16(t.grad) || !aligned16(t.m) || !aligned16(t.v) ||
            (t.param_half && !aligned16(t.param_half)))
            return SNN_ERR_ALIGN;
    }
    // bias corrections and step size in double, handed to the kernel in fp32
    const double lr = hp->lr, b1 = hp->beta1, b2 = hp->beta2;
    const double bc1 = 1.0 - pow(b1, (double)hp->step);
    const double bc2 = 1.0 - pow(b2, (double)hp->step);
    if (!(bc1 > 0.0) || !(bc2 > 0.0)) return SNN_ERR_SHAPE;  // beta = 0 at t = 1 is fine
    AdamwCoef c{};
    c.decay = (float)(1.0 - lr * hp->weight_decay);
    c.beta1 = hp->beta1;
    c.one_minus_beta1 = (float)(1.0 - b1);
    c.beta2 = hp->beta2;
    c.one_minus_beta2 = (float)(1.0 - b2);
    c.step_size = (float)(lr / bc1);
    c.inv_sqrt_bc2 = (float)(1.0 / sqrt(bc2));
    c.eps = hp->eps;
    if (!any) return SNN_OK;
    (void)hipGetLastError();
    return hip_status(launch_adamw(tensors, count, c, stream));
}

}  // extern "C"
