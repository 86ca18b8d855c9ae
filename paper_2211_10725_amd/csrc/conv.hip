// Convolutional synapse of the paper's CSNN (Table I, "5C12-MP2-5C64-MP2"):
// a 5x5 valid cross-correlation, stride 1, plus bias, followed by 2x2 / 2
// max-pooling of the currents before the neuron.
//
// Forward: one lane per pooled current (image, channel, py, px).  It forms
// the four conv outputs of its window, each accumulated in fp32 in the fixed
// order bias, c, ky, kx, so equal receptive fields give bit-equal currents;
// it keeps the first maximum in row-major window order (ties stay with the
// first) and records the choice (0..3) for the backward.  Consecutive lanes
// take consecutive px, so their input patches overlap in cache.
//
// Backward, given dL/dI of the pooled currents:
//   dx[n,c,y,x] = sum_{co,ky,kx} dI[n,co,py,px] w[co,c,ky,kx] over the conv
//                 outputs (y-ky, x-kx) that were selected by their pool window
//                 (gather form, fixed order co, ky, kx: deterministic);
//   dw[co,c,ky,kx] = sum over images and pooled cells of dI times the input
//                 under the selected output, in two passes (per image chunk,
//                 then the chunks in order).
// The bias gradient comes from the neuron scan's per-column sums.
#include "snn_internal.hpp"

namespace snn {
namespace {

constexpr int kThreads = 256;
constexpr int KS = 5;  // kernel size

template <typename TX>
__device__ inline float xval(const TX *x, int64_t i) { return (float)x[i]; }

template <typename TX>
__global__ __launch_bounds__(kThreads) void conv_pool_fwd_kernel(
    int NB, int Ci, int H, int W, int Co, int Hp, int Wp, const TX *__restrict__ x,
    const float *__restrict__ w, const float *__restrict__ bias, float *__restrict__ cur,
    uint8_t *__restrict__ arg) {
    const int64_t idx = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    const int64_t total = (int64_t)NB * Co * Hp * Wp;
    if (idx >= total) return;
    const int px = (int)(idx % Wp);
    const int py = (int)((idx / Wp) % Hp);
    const int co = (int)((idx / ((int64_t)Wp * Hp)) % Co);
    const int64_t nb = idx / ((int64_t)Wp * Hp * Co);
    const float b0 = bias ? bias[co] : 0.f;
    const float *wc = w + (int64_t)co * Ci * KS * KS;
    float v[4];
#pragma unroll
    for (int d = 0; d < 4; ++d) {
        const int oy = 2 * py + (d >> 1), ox = 2 * px + (d & 1);
        float acc = b0;
        for (int c = 0; c < Ci; ++c) {
            const TX *xc = x + ((nb * Ci + c) * H + oy) * W + ox;
            const float *wk = wc + c * KS * KS;
#pragma unroll
            for (int ky = 0; ky < KS; ++ky)
#pragma unroll
                for (int kx = 0; kx < KS; ++kx)
                    acc = __builtin_fmaf(wk[ky * KS + kx], xval<TX>(xc, ky * W + kx), acc);
        }
        v[d] = acc;
    }
    float best = v[0];
    int a = 0;
#pragma unroll
    for (int d = 1; d < 4; ++d)
        if (v[d] > best) {
            best = v[d];
            a = d;
        }
    cur[idx] = best;
    arg[idx] = (uint8_t)a;
}

// dL/dx of the conv input, one lane per input element.
__global__ __launch_bounds__(kThreads) void conv_pool_bwd_dx_kernel(
    int NB, int Ci, int H, int W, int Co, int Hp, int Wp, const float *__restrict__ dI,
    const uint8_t *__restrict__ arg, const float *__restrict__ w, float *__restrict__ dx) {
    const int64_t idx = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    const int64_t total = (int64_t)NB * Ci * H * W;
    if (idx >= total) return;
    const int xx = (int)(idx % W);
    const int yy = (int)((idx / W) % H);
    const int c = (int)((idx / ((int64_t)W * H)) % Ci);
    const int64_t nb = idx / ((int64_t)W * H * Ci);
    float acc = 0.f;
    for (int co = 0; co < Co; ++co) {
        const int64_t pbase = (nb * Co + co) * Hp * Wp;
        const float *wk = w + ((int64_t)co * Ci + c) * KS * KS;
#pragma unroll
        for (int ky = 0; ky < KS; ++ky) {
            const int oy = yy - ky;
            if (oy < 0 || (oy >> 1) >= Hp) continue;
#pragma unroll
            for (int kx = 0; kx < KS; ++kx) {
                const int ox = xx - kx;
                if (ox < 0 || (ox >> 1) >= Wp) continue;
                const int64_t p = pbase + (oy >> 1) * Wp + (ox >> 1);
                if (arg[p] == (uint8_t)(((oy & 1) << 1) | (ox & 1)))
                    acc = __builtin_fmaf(dI[p], wk[ky * KS + kx], acc);
            }
        }
    }
    dx[idx] = acc;
}

// First pass of dL/dw: block (chunk, co); lane j owns weight (c, ky, kx) of
// output channel co and sums over the chunk's images and pooled cells.
template <typename TX>
__global__ __launch_bounds__(kThreads) void conv_pool_bwd_dw_kernel(
    int NB, int Ci, int H, int W, int Co, int Hp, int Wp, int chunk, const float *__restrict__ dI,
    const uint8_t *__restrict__ arg, const TX *__restrict__ x, float *__restrict__ partial) {
    const int co = blockIdx.y;
    const int n0 = blockIdx.x * chunk;
    const int n1 = min(NB, n0 + chunk);
    const int nw = Ci * KS * KS;
    for (int j = threadIdx.x; j < nw; j += kThreads) {
        const int c = j / (KS * KS), ky = (j % (KS * KS)) / KS, kx = j % KS;
        float acc = 0.f;
        for (int nb = n0; nb < n1; ++nb) {
            const int64_t pbase = ((int64_t)nb * Co + co) * Hp * Wp;
            const TX *xc = x + ((int64_t)nb * Ci + c) * H * W;
            for (int p = 0; p < Hp * Wp; ++p) {
                const int a = arg[pbase + p];
                const int oy = 2 * (p / Wp) + (a >> 1), ox = 2 * (p % Wp) + (a & 1);
                acc = __builtin_fmaf(dI[pbase + p], xval<TX>(xc, (oy + ky) * W + ox + kx), acc);
            }
        }
        partial[((int64_t)blockIdx.x * Co + co) * nw + j] = acc;
    }
}

__global__ __launch_bounds__(kThreads) void conv_dw_reduce_kernel(int chunks, int64_t nwt,
                                                                  const float *__restrict__ partial,
                                                                  float *__restrict__ dw) {
    const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (i >= nwt) return;
    float s = 0.f;
    for (int k = 0; k < chunks; ++k) s += partial[(int64_t)k * nwt + i];
    dw[i] = s;
}

int dw_chunks(const ConvGeom &g) {
    // about 64 passes over the weights, at least one image each
    return max(1, min(g.NB, 64));
}

unsigned blocks(int64_t n) { return (unsigned)((n + kThreads - 1) / kThreads); }

}  // namespace

size_t conv_workspace_bytes(const ConvGeom &g, int in_dtype, int w_dtype, int grad_dtype) {
    (void)in_dtype; (void)w_dtype; (void)grad_dtype;
    const int chunks = dw_chunks(g);
    return align_up((size_t)chunks * g.Co * g.Ci * KS * KS * sizeof(float));
}

hipError_t launch_conv_pool_fwd(const ConvGeom &g, const void *x, int in_dtype, const void *w,
                                int w_dtype, const float *bias, float *cur, uint8_t *arg,
                                void *ws, size_t ws_bytes, hipStream_t s) {
    (void)w_dtype; (void)ws; (void)ws_bytes;
    const int64_t total = (int64_t)g.NB * g.Co * g.Hp * g.Wp;
    if (total <= 0) return hipSuccess;
    const float *wf = reinterpret_cast<const float *>(w);
    if (in_dtype == SNN_U8)
        conv_pool_fwd_kernel<uint8_t><<<blocks(total), kThreads, 0, s>>>(
            g.NB, g.Ci, g.H, g.W, g.Co, g.Hp, g.Wp, reinterpret_cast<const uint8_t *>(x), wf, bias,
            cur, arg);
    else
        conv_pool_fwd_kernel<float><<<blocks(total), kThreads, 0, s>>>(
            g.NB, g.Ci, g.H, g.W, g.Co, g.Hp, g.Wp, reinterpret_cast<const float *>(x), wf, bias,
            cur, arg);
    return hipGetLastError();
}

hipError_t launch_conv_pool_bwd(const ConvGeom &g, const void *dcur, int grad_dtype,
                                const uint8_t *arg, const void *x, int in_dtype, const void *w,
                                int w_dtype, float *grad_w, float *grad_x, void *ws,
                                size_t ws_bytes, hipStream_t s) {
    (void)grad_dtype; (void)w_dtype;
    const float *dI = reinterpret_cast<const float *>(dcur);
    const float *wf = reinterpret_cast<const float *>(w);
    if (grad_x) {
        const int64_t total = (int64_t)g.NB * g.Ci * g.H * g.W;
        conv_pool_bwd_dx_kernel<<<blocks(total), kThreads, 0, s>>>(
            g.NB, g.Ci, g.H, g.W, g.Co, g.Hp, g.Wp, dI, arg, wf, grad_x);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (grad_w) {
        const int chunks = dw_chunks(g);
        const int per = (g.NB + chunks - 1) / chunks;
        const int nchunks = (g.NB + per - 1) / per;
        const int64_t nwt = (int64_t)g.Co * g.Ci * KS * KS;
        if (ws == nullptr || ws_bytes < (size_t)nchunks * nwt * sizeof(float))
            return hipErrorInvalidValue;
        float *partial = reinterpret_cast<float *>(ws);
        dim3 grid((unsigned)nchunks, (unsigned)g.Co);
        if (in_dtype == SNN_U8)
            conv_pool_bwd_dw_kernel<uint8_t><<<grid, kThreads, 0, s>>>(
                g.NB, g.Ci, g.H, g.W, g.Co, g.Hp, g.Wp, per, dI, arg,
                reinterpret_cast<const uint8_t *>(x), partial);
        else
            conv_pool_bwd_dw_kernel<float><<<grid, kThreads, 0, s>>>(
                g.NB, g.Ci, g.H, g.W, g.Co, g.Hp, g.Wp, per, dI, arg,
                reinterpret_cast<const float *>(x), partial);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        conv_dw_reduce_kernel<<<blocks(nwt), kThreads, 0, s>>>(nchunks, nwt, partial, grad_w);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace snn
