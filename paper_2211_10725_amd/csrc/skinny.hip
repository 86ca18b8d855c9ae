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
//     A lane owns 4 consecutive n and sums M x 4 products over its rows of a
//     chunk; the 16 waves of a workgroup share the chunk and their sums are
//     added in wave order, the chunks' partial sums then in chunk order.
#include <atomic>

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

// Raw words of 4 consecutive elements of T (1, 2 or 4 words), elements past
// `valid` read as 0; unpacked to floats when they are multiplied.
template <typename T>
struct Raw4 {
    static constexpr int W = sizeof(T);
    uint32_t w[W];
};
template <typename T>
__device__ inline void load_raw4(const T *p, int valid, Raw4<T> &r) {
    if (valid >= 4 && (((uintptr_t)p) & (4 * sizeof(T) - 1)) == 0) {
        if constexpr (sizeof(T) == 4) {
            const uint4 q = *reinterpret_cast<const uint4 *>(p);
            r.w[0] = q.x; r.w[1] = q.y; r.w[2] = q.z; r.w[3] = q.w;
        } else if constexpr (sizeof(T) == 2) {
            const uint2 q = *reinterpret_cast<const uint2 *>(p);
            r.w[0] = q.x; r.w[1] = q.y;
        } else {
            r.w[0] = *reinterpret_cast<const uint32_t *>(p);
        }
    } else {
        T e[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) e[i] = i < valid ? p[i] : T{};
        __builtin_memcpy(r.w, e, sizeof(e));
    }
}
template <typename T>
__device__ inline void unpack4(const Raw4<T> &r, float (&v)[4]) {
    T e[4];
    __builtin_memcpy(e, r.w, sizeof(e));
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = to_f32<T>(e[i]);
}
template <>
__device__ inline void unpack4<uint8_t>(const Raw4<uint8_t> &r, float (&v)[4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = (float)((r.w[0] >> (8 * i)) & 0xffu);  // v_cvt_f32_ubyte
}

// Weight gradient of a layer with few outputs.  A workgroup of 16 waves owns
// one strip of 256 columns (a lane 4 consecutive n) and one chunk of rows.
// The chunk is walked in groups of 16 D rows: the group's small-operand rows
// are staged in LDS, wave w multiplies rows w, w + 16, ... of the group, and
// the next group's big-operand rows are loaded before this group's
// multiply-adds.  At the end the 16 waves' sums are added in wave order
// through LDS; the chunks' partial sums P[chunk][o][n] are added in chunk
// order by the split-K reduction (or written to C when there is one chunk).
constexpr int kFrThreads = 1024;
constexpr int kFrWaves = kFrThreads / 64;

template <typename TA, typename TB, int MP, int D>
struct FewRows {
    static constexpr int G = kFrWaves * D;  // rows per group

    struct Smem {
        float a[G][MP];
        float red[kFrWaves][4][64][4];  // [wave][output of the group of 4][lane][column]
    };

    static __device__ inline void load_rows(const TB *__restrict__ B, int64_t ldb, int g0, int r1,
                                            int wave, int n0, int valid, Raw4<TB> (&x)[D]) {
#pragma unroll
        for (int i = 0; i < D; ++i) {
            const int r = g0 + wave + i * kFrWaves;
            if (r < r1 && valid > 0) load_raw4<TB>(B + (int64_t)r * ldb + n0, valid, x[i]);
            else
#pragma unroll
                for (int w = 0; w < Raw4<TB>::W; ++w) x[i].w[w] = 0u;
        }
    }

    // stage the group's small-operand rows (zeros past the chunk and for o >= M)
    static __device__ inline void stage(const TA *__restrict__ A, int64_t lda, int M, int g0, int r1,
                                        Smem &sm) {
        for (int t = threadIdx.x; t < G * MP; t += kFrThreads) {
            const int i = t / MP, o = t % MP;
            sm.a[i][o] = (g0 + i < r1 && o < M) ? to_f32<TA>(A[(int64_t)(g0 + i) * lda + o]) : 0.f;
        }
    }

    static __device__ inline void multiply(const Smem &sm, int wave, const Raw4<TB> (&x)[D],
                                           float (&acc)[MP][4]) {
#pragma unroll
        for (int i = 0; i < D; ++i) {
            float xv[4];
            unpack4<TB>(x[i], xv);
            const float *ar = sm.a[wave + i * kFrWaves];
#pragma unroll
            for (int q = 0; q < MP / 4; ++q) {
                const float4 a4 = *reinterpret_cast<const float4 *>(ar + 4 * q);
                const float a[4] = {a4.x, a4.y, a4.z, a4.w};
#pragma unroll
                for (int j = 0; j < 4; ++j)
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        acc[4 * q + j][e] = __builtin_fmaf(a[j], xv[e], acc[4 * q + j][e]);
            }
        }
    }
};

template <typename TA, typename TB, int MP, int D>
__global__ __launch_bounds__(kFrThreads) void few_rows_kernel(int M, int N, int R, int rows_per,
                                                              const TA *__restrict__ A, int64_t lda,
                                                              const TB *__restrict__ B, int64_t ldb,
                                                              float *__restrict__ P) {
    using F = FewRows<TA, TB, MP, D>;
    __shared__ __attribute__((aligned(16))) typename F::Smem sm;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int n0 = (blockIdx.x * 64 + lane) * 4;
    const int valid = min(4, N - n0);  // may be <= 0: the lane still joins the staging
    const int r0 = blockIdx.y * rows_per, r1 = min(R, r0 + rows_per);
    float acc[MP][4];
#pragma unroll
    for (int o = 0; o < MP; ++o) acc[o][0] = acc[o][1] = acc[o][2] = acc[o][3] = 0.f;

    Raw4<TB> x0[D], x1[D];
    if (r0 < r1) F::load_rows(B, ldb, r0, r1, wave, n0, valid, x0);
    // two groups per iteration so that both register buffers are named statically
    for (int g0 = r0; g0 < r1; g0 += 2 * F::G) {
        __syncthreads();
        F::stage(A, lda, M, g0, r1, sm);
        __syncthreads();
        const int g1 = g0 + F::G;
        if (g1 < r1) F::load_rows(B, ldb, g1, r1, wave, n0, valid, x1);
        F::multiply(sm, wave, x0, acc);
        if (g1 >= r1) break;
        __syncthreads();
        F::stage(A, lda, M, g1, r1, sm);
        __syncthreads();
        if (g1 + F::G < r1) F::load_rows(B, ldb, g1 + F::G, r1, wave, n0, valid, x0);
        F::multiply(sm, wave, x1, acc);
    }

    // the 16 waves' sums, added in wave order, four outputs at a time
    float *p = P + (int64_t)blockIdx.y * M * N + n0;
#pragma unroll
    for (int og = 0; og < MP / 4; ++og) {
        __syncthreads();
#pragma unroll
        for (int q = 0; q < 4; ++q)
            *reinterpret_cast<float4 *>(sm.red[wave][q][lane]) =
                make_float4(acc[4 * og + q][0], acc[4 * og + q][1], acc[4 * og + q][2],
                            acc[4 * og + q][3]);
        __syncthreads();
        const int o = 4 * og + wave;
        if (wave < 4 && o < M && valid > 0) {
            float s[4] = {0.f, 0.f, 0.f, 0.f};
            for (int w = 0; w < kFrWaves; ++w) {
                const float4 v = *reinterpret_cast<const float4 *>(sm.red[w][wave][lane]);
                s[0] += v.x; s[1] += v.y; s[2] += v.z; s[3] += v.w;
            }
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (e < valid) p[(int64_t)o * N + e] = s[e];
        }
    }
}

unsigned col_blocks(int N) { return (unsigned)((N + 4 * kThreads - 1) / (4 * kThreads)); }

// Chunks of rows for the weight gradient: about one 16-wave workgroup per
// compute unit, each chunk at least one group of rows.
int few_rows_chunks(int N, int R, int group) {
    const int strips = (N + 255) / 256;
    const int per_strip = max(1, (device_cus() + strips - 1) / strips);
    return max(1, min(per_strip, (R + group - 1) / group));
}
constexpr int few_rows_depth(int b_dtype) { return b_dtype == SNN_F32 ? 4 : 8; }

bool a_type_ok(int t) { return t == SNN_F32 || t == SNN_BF16 || t == SNN_F16; }

// The matrix-core variant of the weight gradient: spikes (bytes) against a
// 16-bit or fp32 dL/dI (exact parts, so only when the caller allows them).
bool few_rows_mfma_ok(const GemmArgs &g) {
    return g.allow_split && g.b_dtype == SNN_U8 &&
           (g.a_dtype == SNN_F32 || g.a_dtype == SNN_BF16 || g.a_dtype == SNN_F16);
}

// Chunks of rows: about two workgroups per compute unit, the partial sums
// kept under 8 MiB, at least 32 rows per chunk.
int few_rows_mfma_chunks(int M, int N, int R) {
    const int64_t strips = (N + 511) / 512;
    int64_t S = 2 * (int64_t)device_cus() / strips;
    S = S < ((int64_t)8 << 20) / ((int64_t)M * N * 4) ? S : ((int64_t)8 << 20) / ((int64_t)M * N * 4);
    S = S < (R + 31) / 32 ? S : (R + 31) / 32;
    return S < 1 ? 1 : (int)S;
}



// ---- forward of a layer with few outputs, on the 16-bit matrix cores -------
// C[m][j] = sum_k A[m][k] W[j][k] + bias[j] for j < N <= 16, A (spikes as
// bytes, or fp16) and W (fp32 or fp16) both K-contiguous.  Products are exact
// (a byte is exact in bf16 and fp16; fp32 W is three bf16 parts, fp16 W one
// fp16 part) and accumulate in fp32, as in the general contractions.
//
// One 16x16x32 MFMA tile is 16 rows of A against all (padded) 16 outputs.  W
// is staged once per workgroup into LDS as its parts [part][16][k] (a chunk of
// k at a time when it is long), so it is read from L2 once per compute unit.
// A workgroup of 8 waves covers RWG blocks of 16 rows and splits the k range
// KS = 8 / RWG ways; a wave streams its A fragments (eight k-steps per batch,
// the next batch loaded before this one is multiplied) and the KS partial
// tiles of a row block are added in k order through LDS.
//
// Fragment layout (v_mfma_f32_16x16x32_{bf16,f16}): lane l supplies 8 values
// of row l % 16 of A and of column l % 16 of W at k = 8 (l / 16) + e of the
// step, the same k for both operands; it receives C rows 4 (l / 16) + i,
// column l % 16.
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 half8 __attribute__((ext_vector_type(8)));

constexpr int kNfThreads = 512;
constexpr int kNfWaves = kNfThreads / 64;
constexpr int kNfBatch = 8;  // k-steps of 32 per batch of A loads

__device__ inline uint32_t nf_bf16_bits(float x) {
    const uint32_t b = __float_as_uint(x);
    return (b + 0x7fffu + ((b >> 16) & 1u)) >> 16;
}

// AT: 0 = bytes, 1 = fp16 (A); WP: 3 = fp32 W as bf16 hi/mid/lo, 1 = fp16 W.
template <int AT, int WP>
struct Narrow {
    static constexpr bool F16 = WP == 1;  // MFMA type: fp16 (one part) or bf16
    // k per LDS chunk (a multiple of 64): 99 KB of LDS for fp32 W (the
    // 1000-input readouts in one chunk), 33 KB for fp16 W (several resident
    // workgroups per compute unit for the 4096-input readout); measured best
    static constexpr int KCH = 1024;
    static constexpr int KP = KCH + 8;  // row stride: 16 bytes past a multiple of 128
    static constexpr int AW = AT == 0 ? 2 : 4;  // 32-bit words of an A fragment

    struct Frag { uint32_t w[AW]; };

    // 8 consecutive A values of row m from k (zeros past M and K)
    static __device__ inline void load_a(const void *A, int64_t lda, int M, int K, int m, int k,
                                         bool vec, Frag &f) {
        if (m < M && k + 8 <= K && vec) {
            if constexpr (AT == 0) {
                const uint2 q = *reinterpret_cast<const uint2 *>(
                    reinterpret_cast<const uint8_t *>(A) + (int64_t)m * lda + k);
                f.w[0] = q.x; f.w[1] = q.y;
            } else {
                const uint4 q = *reinterpret_cast<const uint4 *>(
                    reinterpret_cast<const uint16_t *>(A) + (int64_t)m * lda + k);
                f.w[0] = q.x; f.w[1] = q.y; f.w[2] = q.z; f.w[3] = q.w;
            }
        } else {
#pragma unroll
            for (int i = 0; i < AW; ++i) f.w[i] = 0u;
            if (m < M) {
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    if (k + e >= K) continue;
                    if constexpr (AT == 0) {
                        const uint32_t v = reinterpret_cast<const uint8_t *>(A)[(int64_t)m * lda + k + e];
                        f.w[e / 4] |= v << (8 * (e % 4));
                    } else {
                        const uint32_t v = reinterpret_cast<const uint16_t *>(A)[(int64_t)m * lda + k + e];
                        f.w[e / 2] |= v << (16 * (e % 2));
                    }
                }
            }
        }
    }

    // the 8 values as the MFMA's 16-bit operand
    static __device__ inline uint4 to_op(const Frag &f) {
        if constexpr (AT == 1) {
            return make_uint4(f.w[0], f.w[1], f.w[2], f.w[3]);
        } else {
            uint32_t o[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const uint32_t w = f.w[i / 2];
                const float lo = (float)((w >> (16 * (i % 2))) & 0xffu);
                const float hi = (float)((w >> (16 * (i % 2) + 8)) & 0xffu);
                if constexpr (F16) {
                    const _Float16 l = (_Float16)lo, h = (_Float16)hi;  // integers <= 255: exact
                    o[i] = (uint32_t)__builtin_bit_cast(uint16_t, l) |
                           ((uint32_t)__builtin_bit_cast(uint16_t, h) << 16);
                } else {
                    // bytes are exact in bf16: the upper half of the fp32 value
                    o[i] = (__float_as_uint(lo) >> 16) | (__float_as_uint(hi) & 0xffff0000u);
                }
            }
            return make_uint4(o[0], o[1], o[2], o[3]);
        }
    }

    static __device__ inline floatx4 mfma(const uint4 &a, const uint4 &b, const floatx4 &c) {
        if constexpr (F16)
            return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(half8, a),
                                                          __builtin_bit_cast(half8, b), c, 0, 0, 0);
        else
            return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                           __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
    }

    // A fragments of steps sb .. sb + kNfBatch - 1 (zeros from step s1 on)
    static __device__ inline void load_batch(const void *A, int64_t lda, int M, int K, int arow,
                                             int kc0, int kl, int sb, int s1, bool vec,
                                             Frag (&f)[kNfBatch]) {
#pragma unroll
        for (int i = 0; i < kNfBatch; ++i)
            load_a(A, lda, M, sb + i < s1 ? K : 0, arow, kc0 + 32 * (sb + i) + kl, vec, f[i]);
    }

    static __device__ inline void multiply(const uint16_t *Ws, int lane, int kl, int sb, int s1,
                                           const Frag (&f)[kNfBatch], floatx4 &acc) {
#pragma unroll
        for (int i = 0; i < kNfBatch; ++i) {
            if (sb + i < s1) {
                const uint4 a = to_op(f[i]);
#pragma unroll
                for (int p = WP - 1; p >= 0; --p) {  // smallest part first
                    const uint4 b = *reinterpret_cast<const uint4 *>(
                        Ws + (p * 16 + (lane & 15)) * KP + 32 * (sb + i) + kl);
                    acc = mfma(a, b, acc);
                }
            }
        }
    }

    // W[0..16)[kc0 .. kc0 + 32 steps) into LDS as parts (zeros past N and K).
    // A thread owns NQ runs of VE consecutive k: all their global loads are
    // issued before any of them is split and written to LDS.
    static constexpr int VE = WP == 3 ? 4 : 8;  // elements per 16-byte run
    static constexpr int NQ = 16 * KCH / VE / kNfThreads;
    static __device__ inline void stage_w(const void *W, int64_t ldw, bool w_vec, int N, int K,
                                          int kc0, int steps, uint16_t *Ws) {
        const int runs = steps * 32 / VE;  // runs per row of the chunk
        uint4 v[NQ];
#pragma unroll
        for (int i = 0; i < NQ; ++i) {
            const int q = threadIdx.x + i * kNfThreads;
            const int j = q / runs, k = kc0 + (q % runs) * VE;
            v[i] = make_uint4(0u, 0u, 0u, 0u);
            if (j >= N) continue;  // rows N..15 (and runs past the 16 rows) stay zero
            if (w_vec && k + VE <= K) {
                if constexpr (WP == 3)
                    v[i] = *reinterpret_cast<const uint4 *>(reinterpret_cast<const float *>(W) + (int64_t)j * ldw + k);
                else
                    v[i] = *reinterpret_cast<const uint4 *>(reinterpret_cast<const uint16_t *>(W) + (int64_t)j * ldw + k);
            } else {
                uint32_t w[4] = {0u, 0u, 0u, 0u};
#pragma unroll
                for (int e = 0; e < VE; ++e) {
                    if (k + e >= K) continue;
                    if constexpr (WP == 3)
                        w[e] = reinterpret_cast<const uint32_t *>(W)[(int64_t)j * ldw + k + e];
                    else
                        w[e / 2] |= (uint32_t)reinterpret_cast<const uint16_t *>(W)[(int64_t)j * ldw + k + e]
                                    << (16 * (e % 2));
                }
                v[i] = make_uint4(w[0], w[1], w[2], w[3]);
            }
        }
#pragma unroll
        for (int i = 0; i < NQ; ++i) {
            const int q = threadIdx.x + i * kNfThreads;
            const int j = q / runs, k = (q % runs) * VE;
            if (j >= 16) continue;
            if constexpr (WP == 3) {
                const uint32_t x[4] = {v[i].x, v[i].y, v[i].z, v[i].w};
                uint32_t hi[4], mid[4], lo[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float f = __uint_as_float(x[e]);
                    hi[e] = nf_bf16_bits(f);
                    const float r = f - __uint_as_float(hi[e] << 16);
                    mid[e] = nf_bf16_bits(r);
                    lo[e] = nf_bf16_bits(r - __uint_as_float(mid[e] << 16));
                }
                *reinterpret_cast<uint2 *>(Ws + (0 * 16 + j) * KP + k) =
                    make_uint2(hi[0] | (hi[1] << 16), hi[2] | (hi[3] << 16));
                *reinterpret_cast<uint2 *>(Ws + (1 * 16 + j) * KP + k) =
                    make_uint2(mid[0] | (mid[1] << 16), mid[2] | (mid[3] << 16));
                *reinterpret_cast<uint2 *>(Ws + (2 * 16 + j) * KP + k) =
                    make_uint2(lo[0] | (lo[1] << 16), lo[2] | (lo[3] << 16));
            } else {
                *reinterpret_cast<uint4 *>(Ws + j * KP + k) = v[i];
            }
        }
    }
};

template <int AT, int WP>
__global__ __launch_bounds__(kNfThreads) void narrow_fwd_kernel(
    int M, int N, int K, int rwg, const void *__restrict__ A, int64_t lda, bool a_vec,
    const void *__restrict__ W, int64_t ldw, bool w_vec, float *__restrict__ C, int64_t ldc,
    const float *__restrict__ bias) {
    using NF = Narrow<AT, WP>;
    __shared__ __attribute__((aligned(16))) uint16_t Ws[WP * 16 * NF::KP];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int ks = kNfWaves / rwg;
    const int rb = wave % rwg, kq = wave / rwg;
    const int m0 = (blockIdx.x * rwg + rb) * 16;
    const int arow = m0 + (lane & 15), kl = 8 * (lane >> 4);
    floatx4 acc = {0.f, 0.f, 0.f, 0.f};

    for (int kc0 = 0; kc0 < K; kc0 += NF::KCH) {
        const int steps = (min(K - kc0, NF::KCH) + 31) / 32;
        const int per = (steps + ks - 1) / ks;
        const int s0 = min(steps, kq * per), s1 = min(steps, s0 + per);
        typename NF::Frag f0[kNfBatch], f1[kNfBatch];
        if (s0 < s1) NF::load_batch(A, lda, M, K, arow, kc0, kl, s0, s1, a_vec, f0);  // in flight while W is staged
        __syncthreads();  // the previous chunk's reads are done
        NF::stage_w(W, ldw, w_vec, N, K, kc0, steps, Ws);
        __syncthreads();
        for (int sb = s0; sb < s1; sb += 2 * kNfBatch) {
            if (sb + kNfBatch < s1) NF::load_batch(A, lda, M, K, arow, kc0, kl, sb + kNfBatch, s1, a_vec, f1);
            NF::multiply(Ws, lane, kl, sb, s1, f0, acc);
            if (sb + kNfBatch < s1) {
                if (sb + 2 * kNfBatch < s1)
                    NF::load_batch(A, lda, M, K, arow, kc0, kl, sb + 2 * kNfBatch, s1, a_vec, f0);
                NF::multiply(Ws, lane, kl, sb + kNfBatch, s1, f1, acc);
            }
        }
    }

    // add the ks partial tiles of each row block in k order
    __syncthreads();
    float *red = reinterpret_cast<float *>(Ws);  // [wave][4][64]
#pragma unroll
    for (int i = 0; i < 4; ++i) red[(wave * 4 + i) * 64 + lane] = acc[i];
    __syncthreads();
    if (kq != 0) return;
    const int j = lane & 15;
    if (j >= N) return;
    const float bj = bias ? bias[j] : 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int m = m0 + 4 * (lane >> 4) + i;
        float v = 0.f;
        for (int q = 0; q < ks; ++q) v += red[((q * rwg + rb) * 4 + i) * 64 + lane];
        if (m < M) C[(int64_t)m * ldc + j] = v + bj;
    }
}


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
    if (few_rows_mfma_ok(g)) {
        const int S = few_rows_mfma_chunks(g.M, g.N, g.K);
        const int rows_per = (g.K + S - 1) / S;
        const int chunks = (g.K + rows_per - 1) / rows_per;
        return align_up((size_t)chunks * g.M * g.N * sizeof(float));
    }
    const int S = few_rows_chunks(g.N, g.K, kFrWaves * few_rows_depth(g.b_dtype));
    const int rows_per = (g.K + S - 1) / S;
    const int chunks = (g.K + rows_per - 1) / rows_per;
    return align_up((size_t)chunks * g.M * g.N * sizeof(float));
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

template <typename TA, typename TB, int MP>
static void few_rows_launch(const GemmArgs &g, int rows_per, int chunks, float *P, hipStream_t s) {
    constexpr int D = (sizeof(TB) == 4 || MP == 16) ? 4 : 8;
    dim3 grid((unsigned)((g.N + 255) / 256), (unsigned)chunks);
    few_rows_kernel<TA, TB, MP, D><<<grid, kFrThreads, 0, s>>>(
        g.M, g.N, g.K, rows_per, reinterpret_cast<const TA *>(g.A), g.lda,
        reinterpret_cast<const TB *>(g.B), g.ldb, P);
}

template <typename TA, typename TB>
static hipError_t few_rows_typed(const GemmArgs &g, void *ws, size_t ws_bytes, hipStream_t s) {
    const int S = few_rows_chunks(g.N, g.K, kFrWaves * few_rows_depth(g.b_dtype));
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
    if (g.M <= 8) few_rows_launch<TA, TB, 8>(g, rows_per, chunks, P, s);
    else if (g.M <= 12) few_rows_launch<TA, TB, 12>(g, rows_per, chunks, P, s);
    else few_rows_launch<TA, TB, 16>(g, rows_per, chunks, P, s);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || direct) return e;
    return launch_splitk_reduce(g.M, g.N, chunks, P, g.C, g.ldc, g.bias, s);
}

// ---- weight gradient of a layer with few outputs, on the 16-bit matrix cores
// C[o][n] = sum_r A[r][o] X[r][n] for o < M <= 16 with X spikes (bytes) and A
// = dL/dI [rows][M] in fp32 (three exact bf16 parts), bf16 or fp16: the same
// exact products as the general contractions, accumulated in fp32.
//
// One 16x16x32 MFMA tile: the 16 (padded) outputs o against 16 columns, k =
// 32 rows r.  Both operands are stored row-major with r slowest, so neither
// is k-contiguous: a lane loads 8 consecutive bytes (columns n_l .. n_l + 7)
// of each of its 8 rows and regroups them into 8 B fragments, one per column
// offset q; MFMA q of a step covers columns n_w + 8 j + q (j = 0..15), so a
// wave covers 128 columns with 8 MFMAs per part and step.  A's rows of a
// group of 256 are staged in LDS transposed, as parts [part][o][r].  The
// chunks' partial sums P[chunk][o][n] are added by the split-K reduction.
constexpr int kFmThreads = 256;
constexpr int kFmRows = 256;             // rows of a staged group (8 steps of 32)
constexpr int kFmLdr = kFmRows + 8;      // LDS row stride (elements)

template <int AT>  // 0: fp32 A as three bf16 parts, 1: bf16 A, 2: fp16 A (fp16 MFMA)
struct FewRowsMfma {
    static constexpr int NP = AT == 0 ? 3 : 1;
    static constexpr bool F16 = AT == 2;

    // X[r][n .. n + 7] (zeros past R or N)
    static __device__ inline uint2 load_x(const uint8_t *__restrict__ X, int64_t ldx, int r, int r1,
                                          int n, int N, bool vec) {
        if (r >= r1) return make_uint2(0u, 0u);
        const uint8_t *p = X + (int64_t)r * ldx + n;
        if (vec && n + 8 <= N) return *reinterpret_cast<const uint2 *>(p);
        uint32_t w[2] = {0u, 0u};
#pragma unroll
        for (int e = 0; e < 8; ++e)
            if (n + e < N) w[e / 4] |= (uint32_t)p[e] << (8 * (e % 4));
        return make_uint2(w[0], w[1]);
    }

    static __device__ inline void load_step(const uint8_t *__restrict__ X, int64_t ldx, int rs,
                                            int h, int r1, int n, int N, bool vec, uint2 (&x)[8]) {
#pragma unroll
        for (int e = 0; e < 8; ++e) x[e] = load_x(X, ldx, rs + 8 * h + e, r1, n, N, vec);
    }

    // column q of the lane's 8 rows as the MFMA's 16-bit operand (bytes are
    // exact in bf16 and fp16)
    template <int Q>
    static __device__ inline uint4 column(const uint2 (&x)[8]) {
        uint32_t w[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const uint32_t s0 = Q < 4 ? x[2 * i].x : x[2 * i].y;
            const uint32_t s1 = Q < 4 ? x[2 * i + 1].x : x[2 * i + 1].y;
            const float f0 = (float)((s0 >> (8 * (Q % 4))) & 0xffu);
            const float f1 = (float)((s1 >> (8 * (Q % 4))) & 0xffu);
            if constexpr (F16) {
                const _Float16 h0 = (_Float16)f0, h1 = (_Float16)f1;
                w[i] = (uint32_t)__builtin_bit_cast(uint16_t, h0) |
                       ((uint32_t)__builtin_bit_cast(uint16_t, h1) << 16);
            } else {
                w[i] = (__float_as_uint(f0) >> 16) | (__float_as_uint(f1) & 0xffff0000u);
            }
        }
        return make_uint4(w[0], w[1], w[2], w[3]);
    }

    static __device__ inline floatx4 mfma(const uint4 &a, const uint4 &b, const floatx4 &c) {
        if constexpr (F16)
            return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(half8, a),
                                                          __builtin_bit_cast(half8, b), c, 0, 0, 0);
        else
            return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                           __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
    }

    template <int Q>
    static __device__ inline void mult_q(const uint4 (&a)[NP], const uint2 (&x)[8], floatx4 (&acc)[8]) {
        const uint4 b = column<Q>(x);
#pragma unroll
        for (int p = NP - 1; p >= 0; --p) acc[Q] = mfma(a[p], b, acc[Q]);  // smallest part first
    }

    // one step of 32 rows: A fragments from LDS, the 8 column MFMAs
    static __device__ inline void step(const uint16_t *As, int j, int h, int s, const uint2 (&x)[8],
                                       floatx4 (&acc)[8]) {
        uint4 a[NP];
#pragma unroll
        for (int p = 0; p < NP; ++p)
            a[p] = *reinterpret_cast<const uint4 *>(As + (p * 16 + j) * kFmLdr + 32 * s + 8 * h);
        mult_q<0>(a, x, acc); mult_q<1>(a, x, acc); mult_q<2>(a, x, acc); mult_q<3>(a, x, acc);
        mult_q<4>(a, x, acc); mult_q<5>(a, x, acc); mult_q<6>(a, x, acc); mult_q<7>(a, x, acc);
    }

    // A rows g0 .. g0 + kFmRows - 1 (zeros past r1 and for o >= M) as parts
    static __device__ inline void stage(const void *A, int64_t lda, int M, int g0, int r1,
                                        uint16_t *As) {
        for (int t = threadIdx.x; t < kFmRows * 16; t += kFmThreads) {
            const int i = t / 16, o = t % 16, r = g0 + i;
            const bool in = r < r1 && o < M;
            if constexpr (AT == 0) {
                const float v = in ? reinterpret_cast<const float *>(A)[(int64_t)r * lda + o] : 0.f;
                const uint32_t hi = nf_bf16_bits(v);
                const float rr = v - __uint_as_float(hi << 16);
                const uint32_t mid = nf_bf16_bits(rr);
                const uint32_t lo = nf_bf16_bits(rr - __uint_as_float(mid << 16));
                As[(0 * 16 + o) * kFmLdr + i] = (uint16_t)hi;
                As[(1 * 16 + o) * kFmLdr + i] = (uint16_t)mid;
                As[(2 * 16 + o) * kFmLdr + i] = (uint16_t)lo;
            } else {
                As[o * kFmLdr + i] = in ? reinterpret_cast<const uint16_t *>(A)[(int64_t)r * lda + o] : 0;
            }
        }
    }
};

template <int AT>
__global__ __launch_bounds__(kFmThreads) void few_rows_mfma_kernel(
    int M, int N, int R, int rows_per, const void *__restrict__ A, int64_t lda,
    const uint8_t *__restrict__ X, int64_t ldx, bool x_vec, float *__restrict__ P) {
    using F = FewRowsMfma<AT>;
    __shared__ __attribute__((aligned(16))) uint16_t As[F::NP * 16 * kFmLdr];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int h = lane >> 4, j = lane & 15;
    const int n_l = (blockIdx.x * (kFmThreads / 64) + wave) * 128 + 8 * j;
    const int r0 = blockIdx.y * rows_per, r1 = min(R, r0 + rows_per);
    floatx4 acc[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) acc[q] = floatx4{0.f, 0.f, 0.f, 0.f};
    uint2 xa[8], xb[8];
    for (int g0 = r0; g0 < r1; g0 += kFmRows) {
        F::load_step(X, ldx, g0, h, r1, n_l, N, x_vec, xa);  // in flight while A is staged
        __syncthreads();
        F::stage(A, lda, M, g0, r1, As);
        __syncthreads();
        // steps of 32 rows, the next step's rows loaded before this one is multiplied
        for (int s = 0; s < kFmRows / 32 && g0 + 32 * s < r1; s += 2) {
            const bool more = s + 1 < kFmRows / 32 && g0 + 32 * (s + 1) < r1;
            if (more) F::load_step(X, ldx, g0 + 32 * (s + 1), h, r1, n_l, N, x_vec, xb);
            F::step(As, j, h, s, xa, acc);
            if (!more) break;
            if (s + 2 < kFmRows / 32 && g0 + 32 * (s + 2) < r1)
                F::load_step(X, ldx, g0 + 32 * (s + 2), h, r1, n_l, N, x_vec, xa);
            F::step(As, j, h, s + 1, xb, acc);
        }
    }
    // lane: outputs o = 4 h + i, columns n_l + q
    float *p = P + (int64_t)blockIdx.y * M * N;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int o = 4 * h + i;
        if (o >= M) continue;
        float *row = p + (int64_t)o * N + n_l;
        if (n_l + 8 <= N && (((uintptr_t)row) & 15) == 0) {
            *reinterpret_cast<float4 *>(row) = make_float4(acc[0][i], acc[1][i], acc[2][i], acc[3][i]);
            *reinterpret_cast<float4 *>(row + 4) = make_float4(acc[4][i], acc[5][i], acc[6][i], acc[7][i]);
        } else {
#pragma unroll
            for (int q = 0; q < 8; ++q)
                if (n_l + q < N) row[q] = acc[q][i];
        }
    }
}

// Long contractions only: below a few hundred k the per-workgroup staging of
// W and the LDS it holds outweigh the work.
constexpr int kNarrowMinK = 256;

bool narrow_fwd_applies(const GemmArgs &g) {
    if (!(g.N >= 1 && g.N <= 16 && g.M >= 1 && g.K >= kNarrowMinK && g.a_kc && g.b_kc &&
          g.allow_split && g.ldb >= g.K && g.lda >= g.K))
        return false;
    if (g.a_dtype == SNN_U8) return g.b_dtype == SNN_F32 || g.b_dtype == SNN_F16;
    return g.a_dtype == SNN_F16 && g.b_dtype == SNN_F16;
}

// resident workgroups per compute unit of one instance (runtime query, cached per device)
template <int AT, int WP>
int narrow_blocks_per_cu() {
    static std::atomic<int> cache[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 1;
    int v = cache[dev].load(std::memory_order_relaxed);
    if (v == 0) {
        int nb = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
                &nb, reinterpret_cast<const void *>(&narrow_fwd_kernel<AT, WP>), kNfThreads, 0) !=
                hipSuccess || nb <= 0)
            nb = 1;
        v = nb;
        cache[dev].store(v, std::memory_order_relaxed);
    }
    return v;
}

template <int AT, int WP>
static hipError_t narrow_typed(const GemmArgs &g, hipStream_t s) {
    // Row blocks per workgroup: a wave streams 16 x K / (8 / rwg) of A and
    // each workgroup stages all of W; pick the rwg that minimises rounds x
    // (A bytes per wave + W bytes).
    const int blocks = (g.M + 15) / 16;
    const int64_t slots = (int64_t)device_cus() * narrow_blocks_per_cu<AT, WP>();
    const double sa = AT == 0 ? 1.0 : 2.0, sw = WP == 3 ? 4.0 : 2.0;
    int rwg = 8;
    double best = 1e300;
    for (int r = 8; r >= 1; r /= 2) {
        const int64_t wgs = (blocks + r - 1) / r;
        const double cost = (double)((wgs + slots - 1) / slots) * (r * sa / kNfWaves + sw);
        if (cost < best) {
            best = cost;
            rwg = r;
        }
    }
    const unsigned grid = (unsigned)((blocks + rwg - 1) / rwg);
    const bool a_vec = (g.lda % 8) == 0 && (((uintptr_t)g.A) & 15) == 0;
    const bool w_vec = (g.ldb % Narrow<AT, WP>::VE) == 0 && (((uintptr_t)g.B) & 15) == 0;
    narrow_fwd_kernel<AT, WP><<<grid, kNfThreads, 0, s>>>(g.M, g.N, g.K, rwg, g.A, g.lda, a_vec,
                                                          g.B, g.ldb, w_vec, g.C, g.ldc, g.bias);
    return hipGetLastError();
}

hipError_t launch_narrow_fwd(const GemmArgs &g, hipStream_t s) {
    if (g.a_dtype == SNN_F16) return narrow_typed<1, 1>(g, s);
    if (g.b_dtype == SNN_F16) return narrow_typed<0, 1>(g, s);
    return narrow_typed<0, 3>(g, s);
}

template <int AT>
static hipError_t few_rows_mfma_typed(const GemmArgs &g, void *ws, size_t ws_bytes, hipStream_t s) {
    const int S = few_rows_mfma_chunks(g.M, g.N, g.K);
    const int rows_per = (g.K + S - 1) / S;
    const int chunks = (g.K + rows_per - 1) / rows_per;
    const bool direct = chunks == 1 && g.ldc == g.N && g.bias == nullptr;
    float *P = g.C;
    if (!direct) {
        if (ws == nullptr || ws_bytes < (size_t)chunks * g.M * g.N * sizeof(float))
            return hipErrorInvalidValue;
        P = reinterpret_cast<float *>(ws);
    }
    const bool x_vec = (g.ldb % 8) == 0 && (((uintptr_t)g.B) & 7) == 0;
    dim3 grid((unsigned)((g.N + 511) / 512), (unsigned)chunks);
    few_rows_mfma_kernel<AT><<<grid, kFmThreads, 0, s>>>(
        g.M, g.N, g.K, rows_per, g.A, g.lda, reinterpret_cast<const uint8_t *>(g.B), g.ldb, x_vec, P);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || direct) return e;
    return launch_splitk_reduce(g.M, g.N, chunks, P, g.C, g.ldc, g.bias, s);
}

hipError_t launch_few_rows(const GemmArgs &g, void *ws, size_t ws_bytes, hipStream_t s) {
    if (few_rows_mfma_ok(g)) {
        if (g.a_dtype == SNN_F32) return few_rows_mfma_typed<0>(g, ws, ws_bytes, s);
        if (g.a_dtype == SNN_BF16) return few_rows_mfma_typed<1>(g, ws, ws_bytes, s);
        return few_rows_mfma_typed<2>(g, ws, ws_bytes, s);
    }
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
