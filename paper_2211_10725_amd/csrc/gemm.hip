// Synaptic contractions on the gfx950 matrix cores (fp32 MFMA).
//
//   C[M,N] = sum_k A(m,k) B(n,k) (+ bias[n])
//
// covers the three products of a dense layer: currents I = x W^T (+b),
// dW = dI^T x (K = T*B, split over K) and dx = dI W.  Either operand may be
// stored K-contiguous or M/N-contiguous, as fp32, fp16, bf16 or spike bytes;
// tiles are converted to fp32 on the way into LDS (spikes are exact in any
// type) and multiplied with v_mfma_f32_16x16x4_f32, accumulating in fp32.
//
// Workgroup: 256 threads = 4 wave64s, tile BM x BN x 16 staged in LDS in a
// k-major layout so that each MFMA operand fetch is 16 consecutive floats per
// quarter-wave.  The next tile is fetched from global memory into registers
// while the current one is multiplied.  When there are too few output tiles
// to fill the 256 CUs, K is split over blockIdx.z and the partial products are
// summed by a second kernel in fixed split order (deterministic).
#include "snn_internal.hpp"

namespace snn {
namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int BK = 16;

template <typename T>
__device__ inline float to_f32(T v);
template <>
__device__ inline float to_f32<float>(float v) { return v; }
template <>
__device__ inline float to_f32<uint8_t>(uint8_t v) { return (float)v; }
template <>
__device__ inline float to_f32<_Float16>(_Float16 v) { return (float)v; }
struct bf16_t { uint16_t bits; };
template <>
__device__ inline float to_f32<bf16_t>(bf16_t v) { return __uint_as_float((uint32_t)v.bits << 16); }

// Load SEG consecutive elements starting at p, of which the first `valid`
// are in range (the rest read as 0).  Uses 4..16-byte vector loads when the
// whole segment is in range and the address is suitably aligned.
template <typename T, int SEG>
__device__ inline void load_seg(const T *p, int valid, float (&out)[SEG]) {
    constexpr int BYTES = SEG * (int)sizeof(T);
    constexpr int VB = BYTES >= 16 ? 16 : BYTES;  // vector width in bytes
    if (BYTES >= 4 && valid >= SEG && (((uintptr_t)p) & (VB - 1)) == 0) {
        constexpr int PER = VB / (int)sizeof(T);  // elements per vector load
#pragma unroll
        for (int c = 0; c < SEG / PER; ++c) {
            const char *q = reinterpret_cast<const char *>(p + c * PER);
            if constexpr (VB == 16) {
                const uint4 w = *reinterpret_cast<const uint4 *>(q);
                const T *e = reinterpret_cast<const T *>(&w);
#pragma unroll
                for (int i = 0; i < PER; ++i) out[c * PER + i] = to_f32<T>(e[i]);
            } else if constexpr (VB == 8) {
                const uint2 w = *reinterpret_cast<const uint2 *>(q);
                const T *e = reinterpret_cast<const T *>(&w);
#pragma unroll
                for (int i = 0; i < PER; ++i) out[c * PER + i] = to_f32<T>(e[i]);
            } else {
                const uint32_t w = *reinterpret_cast<const uint32_t *>(q);
                const T *e = reinterpret_cast<const T *>(&w);
#pragma unroll
                for (int i = 0; i < PER; ++i) out[c * PER + i] = to_f32<T>(e[i]);
            }
        }
    } else {
#pragma unroll
        for (int i = 0; i < SEG; ++i) out[i] = (i < valid) ? to_f32<T>(p[i]) : 0.f;
    }
}

// Row padding of a k-major LDS tile: a row stride that is 16 mod 64 words puts
// the four k-rows read by one MFMA operand fetch in disjoint bank groups.
constexpr int lds_stride(int R) { return R + ((16 - (R % 64)) % 64 + 64) % 64; }

// Operand tile loader: R rows (M or N) x BK k.  Each thread owns one segment
// of SEG = R*BK/256 elements, contiguous in memory.
template <typename T, bool KC, int R>
struct TileLoader {
    static constexpr int SEG = R * BK / kThreads;
    static_assert(SEG >= 1, "tile too small");
    float v[SEG];
    const T *ptr;
    int valid;
    int lr, lk;  // LDS coordinates of the first element

    __device__ inline void setup(const T *base, int64_t ld, int rows, int row0, int k0, int kend) {
        const int tid = threadIdx.x;
        if constexpr (KC) {
            // consecutive threads take consecutive rows; SEG contiguous k each
            lr = tid % R;
            lk = (tid / R) * SEG;
            const int r = row0 + lr, k = k0 + lk;
            valid = (r < rows) ? max(0, min(SEG, kend - k)) : 0;
            ptr = base + (int64_t)r * ld + k;
        } else {
            // consecutive threads take consecutive row segments of one k-row
            constexpr int per_k = R / SEG;
            lr = (tid % per_k) * SEG;
            lk = tid / per_k;
            const int r = row0 + lr, k = k0 + lk;
            valid = (k < kend) ? max(0, min(SEG, rows - r)) : 0;
            ptr = base + (int64_t)k * ld + r;
        }
    }
    __device__ inline void fetch() {
        if (valid > 0) load_seg<T, SEG>(ptr, valid, v);
        else {
#pragma unroll
            for (int i = 0; i < SEG; ++i) v[i] = 0.f;
        }
    }
    template <int STRIDE>
    __device__ inline void store(float *lds) const {
        if constexpr (KC) {
#pragma unroll
            for (int i = 0; i < SEG; ++i) lds[(lk + i) * STRIDE + lr] = v[i];
        } else {
#pragma unroll
            for (int i = 0; i < SEG; ++i) lds[lk * STRIDE + lr + i] = v[i];
        }
    }
};

template <typename TA, typename TB, bool A_KC, bool B_KC, int BM, int BN, int WAVES_M>
__global__ __launch_bounds__(kThreads) void gemm_f32_kernel(
    int M, int N, int K, int k_chunk, int tiles_n, const TA *__restrict__ A, int64_t lda,
    const TB *__restrict__ B, int64_t ldb, float *__restrict__ C, int64_t ldc,
    int64_t split_stride, const float *__restrict__ bias) {
    constexpr int WAVES_N = 4 / WAVES_M;
    constexpr int WT_M = BM / WAVES_M, WT_N = BN / WAVES_N;
    constexpr int FM = WT_M / 16, FN = WT_N / 16;
    static_assert(FM >= 1 && FN >= 1, "wave tile must hold a 16x16 block");
    constexpr int SA = lds_stride(BM), SB = lds_stride(BN);
    __shared__ float As[BK * SA];
    __shared__ float Bs[BK * SB];

    // Workgroups are dealt round-robin to the 8 XCDs (each with its own L2);
    // renumber them so that each XCD runs a contiguous range of work items,
    // ordered (split, m-tile, n-tile): neighbours share an operand tile.
    const int item = xcd_local_item();
    const int tiles = gridDim.x;
    const int zk = item / tiles, tile = item % tiles;
    const int tm = tile / tiles_n, tn = tile % tiles_n;
    const int m0 = tm * BM, n0 = tn * BN;
    const int kbeg = zk * k_chunk;
    const int kend = min(K, kbeg + k_chunk);

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wm = wave % WAVES_M, wn = wave / WAVES_M;

    floatx4 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

    TileLoader<TA, A_KC, BM> la;
    TileLoader<TB, B_KC, BN> lb;
    if (kbeg < kend) {
        la.setup(A, lda, M, m0, kbeg, kend);
        lb.setup(B, ldb, N, n0, kbeg, kend);
        la.fetch();
        lb.fetch();
    }
    for (int k0 = kbeg; k0 < kend; k0 += BK) {
        __syncthreads();
        la.template store<SA>(As);
        lb.template store<SB>(Bs);
        __syncthreads();
        if (k0 + BK < kend) {
            la.setup(A, lda, M, m0, k0 + BK, kend);
            lb.setup(B, ldb, N, n0, k0 + BK, kend);
            la.fetch();
            lb.fetch();
        }
#pragma unroll
        for (int kk = 0; kk < BK; kk += 4) {
            const int kr = kk + (lane >> 4);
            float a[FM], b[FN];
#pragma unroll
            for (int i = 0; i < FM; ++i) a[i] = As[kr * SA + wm * WT_M + i * 16 + (lane & 15)];
#pragma unroll
            for (int j = 0; j < FN; ++j) b[j] = Bs[kr * SB + wn * WT_N + j * 16 + (lane & 15)];
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], b[j], acc[i][j], 0, 0, 0);
        }
    }

    // D layout of a 16x16 block: lane holds column (lane & 15), rows
    // 4*(lane >> 4) + r for the four accumulator registers r.
    float *Cz = C + (int64_t)zk * split_stride;
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            const int n = n0 + wn * WT_N + j * 16 + (lane & 15);
            if (n >= N) continue;
            const float bn = bias ? bias[n] : 0.f;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int m = m0 + wm * WT_M + i * 16 + 4 * (lane >> 4) + r;
                if (m < M) Cz[(int64_t)m * ldc + n] = acc[i][j][r] + bn;
            }
        }
}

// C[m,n] = sum_{z < S} P[z][m][n] (+ bias[n]), z ascending.
// (divided by the power of two c_div[0] when c_div is set: exact)
__global__ __launch_bounds__(kThreads) void splitk_reduce_kernel(int M, int N, int S,
                                                                 const float *__restrict__ P,
                                                                 float *__restrict__ C, int64_t ldc,
                                                                 const float *__restrict__ bias,
                                                                 const float *__restrict__ c_div) {
    const int64_t total = (int64_t)M * N;
    const int64_t idx = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (idx >= total) return;
    float s = 0.f;
    for (int z = 0; z < S; ++z) s += P[(int64_t)z * total + idx];
    if (c_div) s /= c_div[0];
    const int m = (int)(idx / N), n = (int)(idx % N);
    if (bias) s += bias[n];
    C[(int64_t)m * ldc + n] = s;
}

__global__ __launch_bounds__(kThreads) void divide_kernel(int M, int N, float *__restrict__ C,
                                                          int64_t ldc,
                                                          const float *__restrict__ c_div) {
    const int64_t idx = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (idx >= (int64_t)M * N) return;
    const int m = (int)(idx / N), n = (int)(idx % N);
    C[(int64_t)m * ldc + n] /= c_div[0];
}

// The same sum for many partials (S >= 16): a block reduces 64 outputs, its
// four waves sum fixed quarters of z in ascending order, then the quarters
// are added in order.
__global__ __launch_bounds__(kThreads) void splitk_reduce_wide_kernel(
    int M, int N, int S, const float *__restrict__ P, float *__restrict__ C, int64_t ldc,
    const float *__restrict__ bias, const float *__restrict__ c_div) {
    __shared__ float part[4][64];
    const int64_t total = (int64_t)M * N;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t idx = (int64_t)blockIdx.x * 64 + lane;
    const int per = (S + 3) / 4;
    const int z0 = wave * per, z1 = min(S, z0 + per);
    float s = 0.f;
    if (idx < total) {
#pragma unroll 8
        for (int z = z0; z < z1; ++z) s += P[(int64_t)z * total + idx];
    }
    part[wave][lane] = s;
    __syncthreads();
    if (wave == 0 && idx < total) {
        float r = ((part[0][lane] + part[1][lane]) + part[2][lane]) + part[3][lane];
        if (c_div) r /= c_div[0];
        const int m = (int)(idx / N), n = (int)(idx % N);
        if (bias) r += bias[n];
        C[(int64_t)m * ldc + n] = r;
    }
}

struct Plan {
    int cfg;  // 0: 128x128 (2x2 waves), 1: 64x64 (2x2), 2: 64x16 (4x1), 3: 16x64 (1x4)
    int BM, BN;
    int tiles_m, tiles_n;
    int splits, k_chunk;
};

Plan make_plan(int M, int N, int K) {
    Plan p{};
    if (N <= 16) { p.cfg = 2; p.BM = 64; p.BN = 16; }
    else if (M <= 16) { p.cfg = 3; p.BM = 16; p.BN = 64; }
    else {
        const int64_t big = (int64_t)((M + 127) / 128) * ((N + 127) / 128);
        if (big >= 192) { p.cfg = 0; p.BM = 128; p.BN = 128; }
        else { p.cfg = 1; p.BM = 64; p.BN = 64; }
    }
    p.tiles_m = (M + p.BM - 1) / p.BM;
    p.tiles_n = (N + p.BN - 1) / p.BN;
    const int64_t tiles = (int64_t)p.tiles_m * p.tiles_n;
    const int ksteps = (K + BK - 1) / BK;
    int S = 1;
    if (tiles < 256) {
        S = (int)((512 + tiles - 1) / tiles);
        S = min(S, max(1, ksteps / 8));  // keep at least 8 k-steps per split
        // a small output over a long K (a conv weight gradient) may split
        // further: its partial sums stay small
        S = min(S, (int64_t)M * N <= 65536 ? 256 : 64);
    }
    p.k_chunk = ((ksteps + S - 1) / S) * BK;
    p.splits = (K + p.k_chunk - 1) / p.k_chunk;
    if (p.splits < 1) p.splits = 1;
    return p;
}

template <typename TA, typename TB, bool AK, bool BKc>
void launch_typed(const GemmArgs &g, const Plan &p, float *out, int64_t ldo, int64_t split_stride,
                  const float *bias, hipStream_t s) {
    dim3 grid((unsigned)(p.tiles_m * p.tiles_n), 1, (unsigned)p.splits);
    const TA *A = reinterpret_cast<const TA *>(g.A);
    const TB *B = reinterpret_cast<const TB *>(g.B);
#define SNN_GEMM(BM_, BN_, WM_)                                                              \
    gemm_f32_kernel<TA, TB, AK, BKc, BM_, BN_, WM_><<<grid, kThreads, 0, s>>>(             \
        g.M, g.N, g.K, p.k_chunk, p.tiles_n, A, g.lda, B, g.ldb, out, ldo, split_stride, bias)
    switch (p.cfg) {
        case 0: SNN_GEMM(128, 128, 2); break;
        case 1: SNN_GEMM(64, 64, 2); break;
        case 2: SNN_GEMM(64, 16, 4); break;
        default: SNN_GEMM(16, 64, 1); break;
    }
#undef SNN_GEMM
}

template <typename TA, typename TB>
void launch_layout(const GemmArgs &g, const Plan &p, float *out, int64_t ldo, int64_t ss,
                   const float *bias, hipStream_t s) {
    if (g.a_kc) {
        if (g.b_kc) launch_typed<TA, TB, true, true>(g, p, out, ldo, ss, bias, s);
        else launch_typed<TA, TB, true, false>(g, p, out, ldo, ss, bias, s);
    } else {
        if (g.b_kc) launch_typed<TA, TB, false, true>(g, p, out, ldo, ss, bias, s);
        else launch_typed<TA, TB, false, false>(g, p, out, ldo, ss, bias, s);
    }
}

template <typename TA>
void launch_btype(const GemmArgs &g, const Plan &p, float *out, int64_t ldo, int64_t ss,
                  const float *bias, hipStream_t s) {
    switch (g.b_dtype) {
        case SNN_F32: launch_layout<TA, float>(g, p, out, ldo, ss, bias, s); break;
        case SNN_F16: launch_layout<TA, _Float16>(g, p, out, ldo, ss, bias, s); break;
        case SNN_BF16: launch_layout<TA, bf16_t>(g, p, out, ldo, ss, bias, s); break;
        default: launch_layout<TA, uint8_t>(g, p, out, ldo, ss, bias, s); break;
    }
}

}  // namespace

size_t gemm_workspace_bytes(int M, int N, int K, int a_dtype, int b_dtype, bool a_kc, bool b_kc,
                            bool allow_split) {
    if (M <= 0 || N <= 0 || K <= 0) return 0;
    GemmArgs probe{};
    probe.M = M;
    probe.N = N;
    probe.K = K;
    probe.a_dtype = a_dtype;
    probe.b_dtype = b_dtype;
    probe.a_kc = a_kc;
    probe.b_kc = b_kc;
    probe.allow_split = allow_split;
    probe.lda = a_kc ? K : M;  // densely packed operands (the callers' layouts)
    probe.ldb = b_kc ? K : N;
    if (short_k_applies(probe) || narrow_fwd_applies(probe)) return 0;
    if (few_rows_applies(probe)) return few_rows_workspace_bytes(probe);
    if (gemm_async_applies(probe)) return gemm_async_workspace_bytes(probe);
    if (allow_split && gemm16_applies(probe)) return gemm16_workspace_bytes(probe);
    const Plan p = make_plan(M, N, K);
    if (p.splits <= 1) return 0;
    return align_up((size_t)p.splits * M * N * sizeof(float));
}

namespace {
// a contraction kernel without its own division, then C /= c_div[0] (no bias:
// scaled operands only occur in the backward)
hipError_t divided(hipError_t e, const GemmArgs &g, hipStream_t s) {
    if (e != hipSuccess || g.c_div == nullptr) return e;
    return launch_divide(g.M, g.N, g.C, g.ldc, g.c_div, s);
}
}  // namespace

hipError_t launch_gemm(const GemmArgs &g, void *ws, size_t ws_bytes, hipStream_t s) {
    if (g.M <= 0 || g.N <= 0) return hipSuccess;
    if (g.K <= 0) {
        // empty contraction: C = bias (or 0)
        return hipErrorInvalidValue;
    }
    if (g.c_div && g.bias) return hipErrorInvalidValue;
    if (short_k_applies(g)) return divided(launch_short_k(g, s), g, s);
    if (narrow_fwd_applies(g)) return divided(launch_narrow_fwd(g, s), g, s);
    if (few_rows_applies(g)) return divided(launch_few_rows(g, ws, ws_bytes, s), g, s);
    if (gemm_async_applies(g)) return launch_gemm_async(g, ws, ws_bytes, s);
    if (g.allow_split && gemm16_applies(g)) return divided(launch_gemm16(g, ws, ws_bytes, s), g, s);
    const Plan p = make_plan(g.M, g.N, g.K);
    float *out = g.C;
    int64_t ldo = g.ldc, ss = 0;
    const float *bias = g.bias;
    if (p.splits > 1) {
        if (ws == nullptr || ws_bytes < (size_t)p.splits * g.M * g.N * sizeof(float))
            return hipErrorInvalidValue;
        out = reinterpret_cast<float *>(ws);
        ldo = g.N;
        ss = (int64_t)g.M * g.N;
        bias = nullptr;
    }
    switch (g.a_dtype) {
        case SNN_F32: launch_btype<float>(g, p, out, ldo, ss, bias, s); break;
        case SNN_F16: launch_btype<_Float16>(g, p, out, ldo, ss, bias, s); break;
        case SNN_BF16: launch_btype<bf16_t>(g, p, out, ldo, ss, bias, s); break;
        default: launch_btype<uint8_t>(g, p, out, ldo, ss, bias, s); break;
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (p.splits > 1)
        return launch_splitk_reduce(g.M, g.N, p.splits, out, g.C, g.ldc, g.bias, s, g.c_div);
    return divided(e, g, s);
}

hipError_t launch_splitk_reduce(int M, int N, int S, const float *P, float *C, int64_t ldc,
                                const float *bias, hipStream_t s, const float *c_div) {
    const int64_t total = (int64_t)M * N;
    if (S >= 16)
        splitk_reduce_wide_kernel<<<(unsigned)((total + 63) / 64), kThreads, 0, s>>>(M, N, S, P, C,
                                                                                 ldc, bias, c_div);
    else
        splitk_reduce_kernel<<<(unsigned)((total + kThreads - 1) / kThreads), kThreads, 0, s>>>(
            M, N, S, P, C, ldc, bias, c_div);
    return hipGetLastError();
}

hipError_t launch_divide(int M, int N, float *C, int64_t ldc, const float *c_div, hipStream_t s) {
    const int64_t total = (int64_t)M * N;
    if (total <= 0) return hipSuccess;
    divide_kernel<<<(unsigned)((total + kThreads - 1) / kThreads), kThreads, 0, s>>>(M, N, C, ldc,
                                                                                  c_div);
    return hipGetLastError();
}

}  // namespace snn
