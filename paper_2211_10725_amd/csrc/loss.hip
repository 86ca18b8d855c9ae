// Losses on output spike counts (rate-coded readout: the predicted class is
// the output neuron with the most spikes, Sec. V) and dL/dcounts.
//
// Reductions are fixed-order trees in fp64 (wave64 shuffles, then LDS), so
// the scalar loss is bit-reproducible run to run.
#include "snn_internal.hpp"

namespace snn {
namespace {

constexpr int kThreads = 256;
constexpr int kMsePartials = 1024;  // upper bound on first-pass blocks

__device__ inline double wave_sum(double v) {
    // fixed butterfly order over the 64 lanes of a wave
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

__device__ inline double block_sum(double v) {
    __shared__ double red[kThreads / 64];
    v = wave_sum(v);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (lane == 0) red[wave] = v;
    __syncthreads();
    double s = 0.0;
    if (threadIdx.x == 0) {
        for (int w = 0; w < kThreads / 64; ++w) s += red[w];
    }
    return s;  // valid in thread 0 only
}

// Cross-entropy with the counts as logits, mean over the batch.  One block;
// thread i handles rows i, i+256, ...  A label outside [0, K) makes that
// row's loss and gradient NaN (no out-of-range access).
__global__ __launch_bounds__(kThreads) void ce_kernel(int B, int K, const float *__restrict__ counts,
                                                      const int32_t *__restrict__ labels,
                                                      float *__restrict__ loss,
                                                      float *__restrict__ grad) {
    double part = 0.0;
    const double invB = 1.0 / (double)B;
    for (int b = threadIdx.x; b < B; b += kThreads) {
        const float *c = counts + (int64_t)b * K;
        const int y = labels[b];
        const bool ok = (y >= 0 && y < K);
        double mx = c[0];
        for (int k = 1; k < K; ++k) mx = fmax(mx, (double)c[k]);
        double se = 0.0;
        for (int k = 0; k < K; ++k) se += exp((double)c[k] - mx);
        const double lse = mx + log(se);
        part += ok ? (lse - (double)c[y]) : __builtin_nan("");
        if (grad) {
            for (int k = 0; k < K; ++k) {
                const double p = exp((double)c[k] - mx) / se;
                const double gk = ok ? (p - (k == y ? 1.0 : 0.0)) * invB : __builtin_nan("");
                grad[(int64_t)b * K + k] = (float)gk;
            }
        }
    }
    const double s = block_sum(part);
    if (threadIdx.x == 0) *loss = (float)(s * invB);
}

// Mean squared error, first pass: block z sums (c - y)^2 over its chunk and
// writes the gradient 2 (c - y) / n.
__global__ __launch_bounds__(kThreads) void mse_pass1_kernel(int64_t n, int64_t chunk,
                                                             const float *__restrict__ counts,
                                                             const float *__restrict__ targets,
                                                             float *__restrict__ grad,
                                                             double *__restrict__ partial) {
    const int64_t beg = (int64_t)blockIdx.x * chunk;
    const int64_t end = min(n, beg + chunk);
    const double scale = 2.0 / (double)n;
    double part = 0.0;
    for (int64_t j = beg + threadIdx.x; j < end; j += kThreads) {
        const double d = (double)counts[j] - (double)targets[j];
        part += d * d;
        if (grad) grad[j] = (float)(scale * d);
    }
    const double s = block_sum(part);
    if (threadIdx.x == 0) partial[blockIdx.x] = s;
}

__global__ __launch_bounds__(kThreads) void mse_pass2_kernel(int nparts, int64_t n,
                                                             const double *__restrict__ partial,
                                                             float *__restrict__ loss) {
    double part = 0.0;
    for (int j = threadIdx.x; j < nparts; j += kThreads) part += partial[j];
    const double s = block_sum(part);
    if (threadIdx.x == 0) *loss = (float)(s / (double)n);
}

void mse_shape(int64_t n, int &blocks, int64_t &chunk) {
    int64_t b = (n + 4095) / 4096;
    if (b > kMsePartials) b = kMsePartials;
    if (b < 1) b = 1;
    chunk = (n + b - 1) / b;
    blocks = (int)((n + chunk - 1) / chunk);
}

}  // namespace

size_t loss_workspace_bytes(int kind, int B, int K) {
    if (kind != SNN_LOSS_MSE_COUNT || B <= 0 || K <= 0) return 0;
    int blocks;
    int64_t chunk;
    mse_shape((int64_t)B * K, blocks, chunk);
    return align_up((size_t)blocks * sizeof(double));
}

hipError_t launch_loss(int kind, int B, int K, const float *counts, const int32_t *labels,
                       const float *targets, float *loss, float *grad, void *ws,
                       hipStream_t s) {
    if (kind == SNN_LOSS_CE_COUNT) {
        ce_kernel<<<1, kThreads, 0, s>>>(B, K, counts, labels, loss, grad);
        return hipGetLastError();
    }
    const int64_t n = (int64_t)B * K;
    int blocks;
    int64_t chunk;
    mse_shape(n, blocks, chunk);
    double *partial = reinterpret_cast<double *>(ws);
    mse_pass1_kernel<<<blocks, kThreads, 0, s>>>(n, chunk, counts, targets, grad, partial);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    mse_pass2_kernel<<<1, kThreads, 0, s>>>(blocks, n, partial, loss);
    return hipGetLastError();
}

}  // namespace snn
