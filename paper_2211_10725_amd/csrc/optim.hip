// Fused AdamW weight update for gfx950: every parameter tensor of a network
// in one elementwise pass over HBM (read param, grad, m, v; write param, m, v
// and optionally the fp16 copy the half-precision contractions read).
//
// Work split: a launch takes up to kAdamwMaxTensors (16) tensors by value; each tensor
// is cut into chunks of kChunk elements, one workgroup per chunk, the
// workgroups of tensor i numbered from first_block[i].  A lane handles four
// consecutive elements per iteration (16-byte loads, contiguous across the
// wave) and issues the loads of all its iterations before any arithmetic.
#include "snn_internal.hpp"

namespace snn {
namespace {

constexpr int kThreads = 256;
constexpr int kIters = 4;
constexpr int64_t kChunk = (int64_t)kThreads * 4 * kIters;  // 4096 elements

struct AdamwTensor {
    float *param;
    const float *grad;
    float *m, *v;
    void *half;  // fp16 copy of the updated param, or NULL
    int64_t n;
};

struct AdamwBatch {
    AdamwTensor t[kAdamwMaxTensors];
    int first_block[kAdamwMaxTensors + 1];
    int count;
};

__device__ inline void adamw_element(const AdamwCoef &c, float &p, float g, float &m, float &v) {
    p = p * c.decay;                                   // decoupled weight decay
    m = __builtin_fmaf(c.beta1, m, c.one_minus_beta1 * g);
    v = __builtin_fmaf(c.beta2, v, c.one_minus_beta2 * (g * g));
    const float denom = __builtin_sqrtf(v) * c.inv_sqrt_bc2 + c.eps;  // sqrt(vhat) + eps
    p = p - c.step_size * (m / denom);                  // step_size = lr / (1 - beta1^t)
}

__device__ inline uint16_t to_half_bits(float x) {
    const _Float16 h = (_Float16)x;  // round to nearest even
    return __builtin_bit_cast(uint16_t, h);
}

__global__ __launch_bounds__(kThreads) void adamw_kernel(AdamwBatch b, AdamwCoef c) {
    const int blk = blockIdx.x;
    int ti = 0;
    while (ti + 1 < b.count && blk >= b.first_block[ti + 1]) ++ti;
    const AdamwTensor T = b.t[ti];
    const int64_t base = (int64_t)(blk - b.first_block[ti]) * kChunk;

    float4 P[kIters], G[kIters], M[kIters], V[kIters];
#pragma unroll
    for (int it = 0; it < kIters; ++it) {
        const int64_t i = base + ((int64_t)it * kThreads + threadIdx.x) * 4;
        if (i + 3 < T.n) {
            P[it] = *reinterpret_cast<const float4 *>(T.param + i);
            G[it] = *reinterpret_cast<const float4 *>(T.grad + i);
            M[it] = *reinterpret_cast<const float4 *>(T.m + i);
            V[it] = *reinterpret_cast<const float4 *>(T.v + i);
        }
    }
#pragma unroll
    for (int it = 0; it < kIters; ++it) {
        const int64_t i = base + ((int64_t)it * kThreads + threadIdx.x) * 4;
        if (i + 3 < T.n) {
            adamw_element(c, P[it].x, G[it].x, M[it].x, V[it].x);
            adamw_element(c, P[it].y, G[it].y, M[it].y, V[it].y);
            adamw_element(c, P[it].z, G[it].z, M[it].z, V[it].z);
            adamw_element(c, P[it].w, G[it].w, M[it].w, V[it].w);
            *reinterpret_cast<float4 *>(T.param + i) = P[it];
            *reinterpret_cast<float4 *>(T.m + i) = M[it];
            *reinterpret_cast<float4 *>(T.v + i) = V[it];
            if (T.half) {
                const uint32_t lo = (uint32_t)to_half_bits(P[it].x) |
                                    ((uint32_t)to_half_bits(P[it].y) << 16);
                const uint32_t hi = (uint32_t)to_half_bits(P[it].z) |
                                    ((uint32_t)to_half_bits(P[it].w) << 16);
                *reinterpret_cast<uint2 *>(reinterpret_cast<uint16_t *>(T.half) + i) =
                    make_uint2(lo, hi);
            }
        } else {
            // ragged end of the tensor: at most three elements, one lane
            for (int64_t j = i; j < T.n && j < i + 4; ++j) {
                float p = T.param[j], m = T.m[j], v = T.v[j];
                adamw_element(c, p, T.grad[j], m, v);
                T.param[j] = p;
                T.m[j] = m;
                T.v[j] = v;
                if (T.half) reinterpret_cast<uint16_t *>(T.half)[j] = to_half_bits(p);
            }
        }
    }
}

}  // namespace

int64_t adamw_blocks(int64_t n) { return (n + kChunk - 1) / kChunk; }

hipError_t launch_adamw(const snn_adamw_tensor *t, int count, const AdamwCoef &c, hipStream_t s) {
    int i = 0;
    while (i < count) {
        AdamwBatch b{};
        int blocks = 0;
        int k = 0;
        // fill one launch with up to kAdamwMaxTensors non-empty tensors
        for (; i < count && k < kAdamwMaxTensors; ++i) {
            if (t[i].n <= 0) continue;
            b.t[k] = AdamwTensor{t[i].param, t[i].grad, t[i].m, t[i].v, t[i].param_half, t[i].n};
            b.first_block[k] = blocks;
            blocks += (int)adamw_blocks(t[i].n);
            ++k;
        }
        if (k == 0) break;
        b.first_block[k] = blocks;
        b.count = k;
        adamw_kernel<<<blocks, kThreads, 0, s>>>(b, c);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace snn
