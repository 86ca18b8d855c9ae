// Losses on output spike counts (rate-coded readout: the predicted class is
// the output neuron with the most spikes, Sec. V) and dL/dcounts.  With a
// population code (Sec. V) each class owns P consecutive output neurons and
// the loss is taken on the class counts, the sums over each population; every
// neuron of a population receives its class's gradient.
//
// Reductions are fixed-order trees in fp64 (wave64 shuffles, then LDS), so
// the scalar loss is bit-reproducible run to run.
#include <atomic>

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

// class count k of a row: the sum of its population (exact in fp64)
__device__ inline double class_count(const float *c, int k, int P) {
    double s = 0.0;
    for (int p = 0; p < P; ++p) s += (double)c[(int64_t)k * P + p];
    return s;
}

__device__ inline double wave_max(double v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v = fmax(v, __shfl_xor(v, off, 64));
    return v;
}

// Cross-entropy with the class counts as logits, one wave per row.  Rows of
// up to LDSROW counts are staged in the wave's LDS buffers with coalesced
// loads; lane l sums the populations of classes l, l+64, ... once, max and
// sum of exponentials are wave reductions in a fixed butterfly order, and the
// per-class gradient is written back to the row's K*P neurons with coalesced
// stores.  Longer rows read the counts from global memory.  Returns the
// row's loss (fp64) in every lane.  A label outside [0, K) makes that row's
// loss and gradient NaN (no out-of-range access).
template <int LDSROW>
__device__ inline double ce_row(int b, int B, int K, int P, int lane, const float *__restrict__ counts,
                                const int32_t *__restrict__ labels, float *__restrict__ grad,
                                float *rowbuf, double *cls) {
    const int64_t row = (int64_t)K * P;
    const bool staged = row <= LDSROW;
    const float *cg = counts + (int64_t)b * row;
    if (staged) {
        for (int j = lane; j < (int)row; j += 64) rowbuf[j] = cg[j];
        // read back by other lanes of the same wave: a wave's LDS accesses
        // complete in order, so only the compiler must keep the order
        __builtin_amdgcn_wave_barrier();
        for (int k = lane; k < K; k += 64) cls[k] = class_count(rowbuf, k, P);
        __builtin_amdgcn_wave_barrier();
    }
    const int y = labels[b];
    const bool ok = (y >= 0 && y < K);
    double mx = -__builtin_inf();
    for (int k = lane; k < K; k += 64) mx = fmax(mx, staged ? cls[k] : class_count(cg, k, P));
    mx = wave_max(mx);
    double se = 0.0;
    for (int k = lane; k < K; k += 64) se += exp((staged ? cls[k] : class_count(cg, k, P)) - mx);
    se = wave_sum(se);
    const double invB = 1.0 / (double)B;
    float *gr = grad ? grad + (int64_t)b * row : nullptr;
    if (gr && staged) {
        // per-class gradient in place of the class counts, then spread over
        // each population with coalesced stores
        for (int k = lane; k < K; k += 64) {
            const double p = exp(cls[k] - mx) / se;
            rowbuf[k] = ok ? (float)((p - (k == y ? 1.0 : 0.0)) * invB) : __builtin_nanf("");
        }
        __builtin_amdgcn_wave_barrier();
        for (int j = lane; j < (int)row; j += 64) gr[j] = rowbuf[j / P];
        __builtin_amdgcn_wave_barrier();  // the buffers are reused by the next row
    } else if (gr) {
        for (int k = lane; k < K; k += 64) {
            const double p = exp(class_count(cg, k, P) - mx) / se;
            const double gk = ok ? (p - (k == y ? 1.0 : 0.0)) * invB : __builtin_nan("");
            for (int q = 0; q < P; ++q) gr[(int64_t)k * P + q] = (float)gk;
        }
    }
    const double cy = ok ? (staged ? cls[y] : class_count(cg, y, P)) : 0.0;
    return ok ? (mx + log(se)) - cy : __builtin_nan("");
}

// Rows spread over workgroups (4 rows each); the row losses go to
// partial[b] (fp64), summed in fixed order by ce_sum_kernel.
constexpr int kCeRowLds = 1024;
constexpr int kRowsPerBlock = kThreads / 64;
__global__ __launch_bounds__(kThreads) void ce_rows_kernel(int B, int K, int P,
                                                           const float *__restrict__ counts,
                                                           const int32_t *__restrict__ labels,
                                                           float *__restrict__ grad,
                                                           double *__restrict__ partial) {
    __shared__ float rowbuf[kRowsPerBlock][kCeRowLds];
    __shared__ double cls[kRowsPerBlock][kCeRowLds];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int b = blockIdx.x * kRowsPerBlock + wave;
    if (b >= B) return;  // no workgroup barrier follows
    const double l = ce_row<kCeRowLds>(b, B, K, P, lane, counts, labels, grad, rowbuf[wave], cls[wave]);
    if (lane == 0) partial[b] = l;
}

// loss = sum_b partial[b] / B, fixed order (strided per thread, then tree)
__global__ __launch_bounds__(kThreads) void ce_sum_kernel(int B, const double *__restrict__ partial,
                                                          float *__restrict__ loss) {
    double part = 0.0;
    for (int b = threadIdx.x; b < B; b += kThreads) part += partial[b];
    const double s = block_sum(part);
    if (threadIdx.x == 0) *loss = (float)(s / (double)B);
}

// Small readouts (at most 16 classes, 128 rows and 12288 counts): one
// workgroup stages every count and label in LDS with coalesced loads, then
// each 16-lane group takes rows g, g + 64, ... with one class per lane.  The
// group's butterfly reductions combine the same values in the same tree as
// ce_row's wave-wide ones (there the other lanes add exact zeros, or -inf to
// the maximum), and the row losses are summed in ce_sum_kernel's fixed order,
// so the results equal the two-launch path's bit for bit: one launch whose
// rows are all in flight at once.
constexpr int kCeGroup = 16;
constexpr int kCeSmallThreads = 1024;
constexpr int kCeSmallElems = 12288;
constexpr int kCeSmallMaxB = 128;  // more rows run faster over many workgroups

__device__ inline double group_sum(double v) {
#pragma unroll
    for (int off = kCeGroup / 2; off >= 1; off >>= 1) v += __shfl_xor(v, off, kCeGroup);
    return v;
}

__device__ inline double group_max(double v) {
#pragma unroll
    for (int off = kCeGroup / 2; off >= 1; off >>= 1) v = fmax(v, __shfl_xor(v, off, kCeGroup));
    return v;
}

__global__ __launch_bounds__(kCeSmallThreads) void ce_small_kernel(int B, int K, int P,
                                                                   const float *__restrict__ counts,
                                                                   const int32_t *__restrict__ labels,
                                                                   float *__restrict__ grad,
                                                                   float *__restrict__ loss) {
    __shared__ float cnt[kCeSmallElems];
    __shared__ int32_t lab[kCeSmallMaxB];
    __shared__ double part[kCeSmallMaxB];
    __shared__ double red[kThreads / 64];
    const int row = K * P, n = B * row;
    for (int i = threadIdx.x; i < n; i += kCeSmallThreads) cnt[i] = counts[i];
    for (int b = threadIdx.x; b < B; b += kCeSmallThreads) lab[b] = labels[b];
    __syncthreads();
    const int sub = threadIdx.x % kCeGroup, grp = threadIdx.x / kCeGroup;
    constexpr int G = kCeSmallThreads / kCeGroup;
    const double invB = 1.0 / (double)B;
    for (int b = grp; b < B; b += G) {
        float *rb = cnt + b * row;
        const bool has = sub < K;
        const double c = has ? class_count(rb, sub, P) : 0.0;
        const int y = lab[b];
        const bool ok = (y >= 0 && y < K);
        const double mx = group_max(has ? c : -__builtin_inf());
        const double e = has ? exp(c - mx) : 0.0;
        const double se = group_sum(e);
        const double cy = __shfl(c, ok ? y : 0, kCeGroup);
        if (grad) {
            // the class gradient replaces the class's first count (every
            // count of the row has been read), then spreads over its population
            __builtin_amdgcn_wave_barrier();
            if (has) {
                const double p = e / se;  // e is exp(c - mx), as ce_row recomputes it
                rb[sub] = ok ? (float)((p - (sub == y ? 1.0 : 0.0)) * invB) : __builtin_nanf("");
            }
            __builtin_amdgcn_wave_barrier();
            float *gr = grad + (int64_t)b * row;
            for (int j = sub; j < row; j += kCeGroup) gr[j] = rb[j / P];
        }
        if (sub == 0) part[b] = ok ? (mx + log(se)) - cy : __builtin_nan("");
    }
    __syncthreads();
    // the order of ce_sum_kernel: thread t sums rows t, t + 256, ...; the
    // 256 sums in 4 waves by butterfly, the waves in order
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    double s = 0.0;
    if (threadIdx.x < kThreads)
        for (int b = threadIdx.x; b < B; b += kThreads) s += part[b];
    s = wave_sum(s);
    if (lane == 0 && wave < kThreads / 64) red[wave] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
        double t = 0.0;
        for (int w = 0; w < kThreads / 64; ++w) t += red[w];
        *loss = (float)(t / (double)B);
    }
}

// Mean squared error, first pass: block z sums (c - y)^2 over its chunk of
// the n = B K class entries and writes the gradient 2 (c - y) / n to each
// neuron of the class's population.
__global__ __launch_bounds__(kThreads) void mse_pass1_kernel(int64_t n, int64_t chunk, int P,
                                                             const float *__restrict__ counts,
                                                             const float *__restrict__ targets,
                                                             float *__restrict__ grad,
                                                             double *__restrict__ partial) {
    const int64_t beg = (int64_t)blockIdx.x * chunk;
    const int64_t end = min(n, beg + chunk);
    const double scale = 2.0 / (double)n;
    double part = 0.0;
    for (int64_t j = beg + threadIdx.x; j < end; j += kThreads) {
        // class entry j owns neurons j*P .. j*P + P - 1 of the [B, K*P] counts
        const double d = class_count(counts + j * P, 0, P) - (double)targets[j];
        part += d * d;
        if (grad)
            for (int q = 0; q < P; ++q) grad[j * P + q] = (float)(scale * d);
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
    if (B <= 0 || K <= 0) return 0;
    if (kind == SNN_LOSS_CE_COUNT) return align_up((size_t)B * sizeof(double));  // row losses
    int blocks;
    int64_t chunk;
    mse_shape((int64_t)B * K, blocks, chunk);
    return align_up((size_t)blocks * sizeof(double));
}

hipError_t launch_loss(int kind, int B, int K, int P, const float *counts,
                       const int32_t *labels, const float *targets, float *loss, float *grad,
                       void *ws, hipStream_t s) {
    if (kind == SNN_LOSS_CE_COUNT) {
        if (K <= kCeGroup && B <= kCeSmallMaxB && (int64_t)B * K * P <= kCeSmallElems) {
            ce_small_kernel<<<1, kCeSmallThreads, 0, s>>>(B, K, P, counts, labels, grad, loss);
            return hipGetLastError();
        }
        double *partial = reinterpret_cast<double *>(ws);
        ce_rows_kernel<<<(B + kRowsPerBlock - 1) / kRowsPerBlock, kThreads, 0, s>>>(
            B, K, P, counts, labels, grad, partial);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        ce_sum_kernel<<<1, kThreads, 0, s>>>(B, partial, loss);
        return hipGetLastError();
    }
    const int64_t n = (int64_t)B * K;
    int blocks;
    int64_t chunk;
    mse_shape(n, blocks, chunk);
    double *partial = reinterpret_cast<double *>(ws);
    mse_pass1_kernel<<<blocks, kThreads, 0, s>>>(n, chunk, P, counts, targets, grad, partial);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    mse_pass2_kernel<<<1, kThreads, 0, s>>>(blocks, n, partial, loss);
    return hipGetLastError();
}

// ---- scratch for callers that cannot allocate ------------------------------
// The loss's partial sums (one double per row for cross-entropy, one per
// first-pass block for MSE) in a file-scope device array instead of a
// caller's workspace.  Every device the library runs on holds its own copy
// until the process ends; its address differs per device and is looked up
// once per device with that device current.  Each partial is written before
// it is read, so nothing needs clearing between calls; calls that overlap on
// one device share the array and race.
static __device__ __align__(256) unsigned char scratch[kLossScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::atomic<void *> scratch_ptr[kMaxDevices];
}  // namespace

hipError_t loss_static_scratch(void **ptr) {
    *ptr = nullptr;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    void *p = scratch_ptr[dev].load(std::memory_order_acquire);
    if (p == nullptr) {
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (p == nullptr) return hipErrorInvalidSymbol;
        scratch_ptr[dev].store(p, std::memory_order_release);
    }
    *ptr = p;
    return hipSuccess;
}

}  // namespace snn
