// Contractions of a layer with few outputs (the 10-neuron readout of the
// benchmark networks), where one side of the product is at most 16 wide and
// a matrix-core tile would be mostly empty.  Both kernels are bound by
// streaming the big operand through HBM and run on the vector ALUs with fp32
// fused multiply-adds in a fixed order (deterministic; every product of the
// operand types used here is exact in fp32).
//
//   input gradient, short contraction (K <= 16):
//     C[m][n] = sum_{k<K} A[m][k] B[k][n],  B with n contiguous.
//     A lane owns 4 consecutive n and keeps B[0..K)[n..n+3] in registers; it
//     walks a chunk of rows, reading row m of A at a wave-uniform address.
//   weight gradient, few rows (M <= 16):
//     C[o][n] = sum_r A[r][o] B[r][n]  (A = dL/dI [rows][M], B = x [rows][N]).
//     A lane owns 4 consecutive n and sums M x 4 products over a chunk of
//     rows; the chunks' partial sums are then added in chunk order.
#include "snn_internal.hpp"

namespace snn {
namespace {

constexpr int kThreads = 256;
constexpr int kSkinny = 16;

struct bf16_t {
    uint16_t bits;
};
template <typename T>
__device__ inline float to_f32(T v) { return (float)v; }
template <>
__device__ inline float to_f32<bf16_t>(bf16_t v) { return __uint_as_float((uint32_t)v.bits << 16); }

// 4 consecutive elements as floats, of which the first `valid` are in range
// (the rest read as 0).
template <typename T>
__device__ inline void load4(const T *p, int valid, float (&v)[4]) {
    if (valid >= 4 && (((uintptr_t)p) & (4 * sizeof(T) - 1)) == 0) {
        if constexpr (sizeof(T) == 4) {
            const float4 q = *reinterpret_cast<const float4 *>(p);
            v[0] = q.x; v[1] = q.y; v[2] = q.z; v[3] = q.w;
        } else if constexpr (sizeof(T) == 2) {
            const uint2 q = *reinterpret_cast<const uint2 *>(p);
            const T *h = reinterpret_cast<const T *>(&q);
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = to_f32<T>(h[e]);
        } else {
            const uint32_t q = *reinterpret_cast<const uint32_t *>(p);
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = (float)((q >> (8 * e)) & 0xffu);
        }
    } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = e < valid ? to_f32<T>(p[e]) : 0.f;
    }
}

constexpr int kRowGroup = 32;  // rows whose small operand is staged in LDS at once

// The small operand of kRowGroup rows, [row][k] with k < K <= 16, staged in
// LDS by one coalesced cooperative load; k >= K and rows past `rows` are 0,
// so the multiply-adds below run over all 16 k without branches (adding exact
// zeros) and read a row with four 16-byte LDS reads.
template <typename TA>
__device__ inline void stage_rows(const TA *__restrict__ A, int64_t lda, int K, int r0, int rows,
                                  float (&S)[kRowGroup][kSkinny]) {
    for (int t = threadIdx.x; t < kRowGroup * kSkinny; t += kThreads) {
        const int r = t / kSkinny, k = t % kSkinny;
        S[r][k] = (r0 + r < rows && k < K) ? to_f32<TA>(A[(int64_t)(r0 + r) * lda + k]) : 0.f;
    }
}

__device__ inline void lds_row(const float (&S)[kRowGroup][kSkinny], int r, float (&v)[kSkinny]) {
#pragma unroll
    for (int q = 0; q < kSkinny / 4; ++q) {
        const float4 x = *reinterpret_cast<const float4 *>(&S[r][4 * q]);
        v[4 * q] = x.x; v[4 * q + 1] = x.y; v[4 * q + 2] = x.z; v[4 * q + 3] = x.w;
    }
}

template <typename TA, typename TB>
__global__ __launch_bounds__(kThreads) void short_k_kernel(int M, int N, int K,
                                                           const TA *__restrict__ A, int64_t lda,
                                                           const TB *__restrict__ B, int64_t ldb,
                                                           float *__restrict__ C, int64_t ldc,
                                                           const float *__restrict__ bias) {
    __shared__ __attribute__((aligned(16))) float As[kRowGroup][kSkinny];
    const int n0 = (blockIdx.x * kThreads + threadIdx.x) * 4;
    const int valid = min(4, N - n0);  // may be <= 0: the lane still joins the staging
    float b[kSkinny][4];
#pragma unroll
    for (int k = 0; k < kSkinny; ++k) {
        if (k < K && valid > 0) load4<TB>(B + (int64_t)k * ldb + n0, valid, b[k]);
        else b[k][0] = b[k][1] = b[k][2] = b[k][3] = 0.f;
    }
    float bn[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) bn[e] = (bias && e < valid) ? bias[n0 + e] : 0.f;
    for (int m0 = blockIdx.y * kRowGroup; m0 < M; m0 += gridDim.y * kRowGroup) {
        __syncthreads();
        stage_rows<TA>(A, lda, K, m0, M, As);
        __syncthreads();
        if (valid <= 0) continue;
        const int rows = min(kRowGroup, M - m0);
        for (int r = 0; r < rows; ++r) {
            float a[kSkinny];
            lds_row(As, r, a);
            float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int k = 0; k < kSkinny; ++k)
#pragma unroll
                for (int e = 0; e < 4; ++e) acc[e] = __builtin_fmaf(a[k], b[k][e], acc[e]);
            float *c = C + (int64_t)(m0 + r) * ldc + n0;
            if (valid == 4 && (((uintptr_t)c) & 15) == 0) {
                *reinterpret_cast<float4 *>(c) =
                    make_float4(acc[0] + bn[0], acc[1] + bn[1], acc[2] + bn[2], acc[3] + bn[3]);
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (e < valid) c[e] = acc[e] + bn[e];
            }
        }
    }
}

template <typename TA, typename TB>
__global__ __launch_bounds__(kThreads) void few_rows_kernel(int M, int N, int R, int rows_per,
                                                            const TA *__restrict__ A, int64_t lda,
                                                            const TB *__restrict__ B, int64_t ldb,
                                                            float *__restrict__ P) {
    __shared__ __attribute__((aligned(16))) float As[kRowGroup][kSkinny];
    const int n0 = (blockIdx.x * kThreads + threadIdx.x) * 4;
    const int valid = min(4, N - n0);  // may be <= 0: the lane still joins the staging
    float acc[kSkinny][4];
#pragma unroll
    for (int o = 0; o < kSkinny; ++o) acc[o][0] = acc[o][1] = acc[o][2] = acc[o][3] = 0.f;
    const int r0 = blockIdx.y * rows_per, r1 = min(R, r0 + rows_per);
    for (int g0 = r0; g0 < r1; g0 += kRowGroup) {
        __syncthreads();
        stage_rows<TA>(A, lda, M, g0, r1, As);
        __syncthreads();
        if (valid <= 0) continue;
        const int rows = min(kRowGroup, r1 - g0);
        for (int rb = 0; rb < rows; rb += 8) {
            // 8 rows of the big operand in flight before their multiply-adds
            float x[8][4];
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                if (rb + i < rows) load4<TB>(B + (int64_t)(g0 + rb + i) * ldb + n0, valid, x[i]);
                else x[i][0] = x[i][1] = x[i][2] = x[i][3] = 0.f;
            }
            // rows past the group and outputs o >= M multiply staged zeros
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                float a[kSkinny];
                lds_row(As, rb + i, a);
#pragma unroll
                for (int o = 0; o < kSkinny; ++o)
#pragma unroll
                    for (int e = 0; e < 4; ++e) acc[o][e] = __builtin_fmaf(a[o], x[i][e], acc[o][e]);
            }
        }
    }
    if (valid <= 0) return;
    // partial sums of this chunk: P[chunk][o][n]
    float *p = P + (int64_t)blockIdx.y * M * N + n0;
#pragma unroll
    for (int o = 0; o < kSkinny; ++o)
        if (o < M)
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (e < valid) p[(int64_t)o * N + e] = acc[o][e];
}

unsigned col_blocks(int N) { return (unsigned)((N + 4 * kThreads - 1) / (4 * kThreads)); }

// chunks of rows for the weight gradient: about 1024 workgroups, >= 16 rows each
int few_rows_chunks(int N, int R) {
    const int per_col = max(1, 1024 / (int)col_blocks(N));
    return max(1, min(per_col, (R + 15) / 16));
}

bool a_type_ok(int t) { return t == SNN_F32 || t == SNN_BF16 || t == SNN_F16; }

}  // namespace

// Below about 4M elements of the large operand, launch latency dominates and
// the general kernels (one launch fewer) are as fast (measured on MI355X).
constexpr double kSkinnyMinElems = 4194304.0;

bool short_k_applies(const GemmArgs &g) {
    return g.K >= 1 && g.K <= kSkinny && g.a_kc && !g.b_kc && a_type_ok(g.a_dtype) &&
           (g.b_dtype == SNN_F32 || g.b_dtype == SNN_F16) &&
           (double)g.M * g.N >= kSkinnyMinElems;
}

bool few_rows_applies(const GemmArgs &g) {
    return g.M >= 1 && g.M <= kSkinny && !g.a_kc && !g.b_kc && a_type_ok(g.a_dtype) &&
           (g.b_dtype == SNN_U8 || g.b_dtype == SNN_F16 || g.b_dtype == SNN_F32) &&
           (double)g.K * g.N >= kSkinnyMinElems;
}

size_t few_rows_workspace_bytes(const GemmArgs &g) {
    if (!few_rows_applies(g) || g.K <= 0) return 0;
    return align_up((size_t)few_rows_chunks(g.N, g.K) * g.M * g.N * sizeof(float));
}

template <typename TA, typename TB>
static hipError_t short_k_typed(const GemmArgs &g, hipStream_t s) {
    // one row group per workgroup (grid-stride beyond 65535 groups)
    const int groups = (g.M + kRowGroup - 1) / kRowGroup;
    dim3 grid(col_blocks(g.N), (unsigned)min(groups, 65535));
    short_k_kernel<TA, TB><<<grid, kThreads, 0, s>>>(
        g.M, g.N, g.K, reinterpret_cast<const TA *>(g.A), g.lda,
        reinterpret_cast<const TB *>(g.B), g.ldb, g.C, g.ldc, g.bias);
    return hipGetLastError();
}

hipError_t launch_short_k(const GemmArgs &g, hipStream_t s) {
    const bool bf = g.b_dtype == SNN_F32;
    switch (g.a_dtype) {
        case SNN_F32: return bf ? short_k_typed<float, float>(g, s) : short_k_typed<float, _Float16>(g, s);
        case SNN_BF16: return bf ? short_k_typed<bf16_t, float>(g, s) : short_k_typed<bf16_t, _Float16>(g, s);
        default: return bf ? short_k_typed<_Float16, float>(g, s) : short_k_typed<_Float16, _Float16>(g, s);
    }
}

template <typename TA, typename TB>
static hipError_t few_rows_typed(const GemmArgs &g, void *ws, size_t ws_bytes, hipStream_t s) {
    const int S = few_rows_chunks(g.N, g.K);
    const int rows_per = (g.K + S - 1) / S;
    const int chunks = (g.K + rows_per - 1) / rows_per;
    // one chunk writes C directly when it is densely packed and has no bias
    const bool direct = chunks == 1 && g.ldc == g.N && g.bias == nullptr;
    float *P = g.C;
    if (!direct) {
        if (ws == nullptr || ws_bytes < (size_t)chunks * g.M * g.N * sizeof(float))
            return hipErrorInvalidValue;
        P = reinterpret_cast<float *>(ws);
    }
    dim3 grid(col_blocks(g.N), (unsigned)chunks);
    few_rows_kernel<TA, TB><<<grid, kThreads, 0, s>>>(
        g.M, g.N, g.K, rows_per, reinterpret_cast<const TA *>(g.A), g.lda,
        reinterpret_cast<const TB *>(g.B), g.ldb, P);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || direct) return e;
    return launch_splitk_reduce(g.M, g.N, chunks, P, g.C, g.ldc, g.bias, s);
}

hipError_t launch_few_rows(const GemmArgs &g, void *ws, size_t ws_bytes, hipStream_t s) {
    switch (g.a_dtype) {
        case SNN_F32:
            if (g.b_dtype == SNN_U8) return few_rows_typed<float, uint8_t>(g, ws, ws_bytes, s);
            if (g.b_dtype == SNN_F16) return few_rows_typed<float, _Float16>(g, ws, ws_bytes, s);
            return few_rows_typed<float, float>(g, ws, ws_bytes, s);
        case SNN_BF16:
            if (g.b_dtype == SNN_U8) return few_rows_typed<bf16_t, uint8_t>(g, ws, ws_bytes, s);
            if (g.b_dtype == SNN_F16) return few_rows_typed<bf16_t, _Float16>(g, ws, ws_bytes, s);
            return few_rows_typed<bf16_t, float>(g, ws, ws_bytes, s);
        default:
            if (g.b_dtype == SNN_U8) return few_rows_typed<_Float16, uint8_t>(g, ws, ws_bytes, s);
            if (g.b_dtype == SNN_F16) return few_rows_typed<_Float16, _Float16>(g, ws, ws_bytes, s);
            return few_rows_typed<_Float16, float>(g, ws, ws_bytes, s);
    }
}

}  // namespace snn
