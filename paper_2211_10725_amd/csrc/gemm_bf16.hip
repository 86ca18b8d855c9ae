// Spike x fp32 contractions on the bf16 matrix cores, exact products.
//
// A spike (0/1, or any byte value) is exact in bf16.  An fp32 value x splits
// exactly into three bf16 parts, x = hi + mid + lo: hi = bf16(x) (round to
// nearest even), mid = bf16(x - hi), lo = x - hi - mid; each subtraction is
// exact (the operands are within a factor of two, Sterbenz), x - hi has at
// most 16 significant bits and x - hi - mid at most 8, so lo is exact in bf16
// (down to the bottom of the fp32 normal range).  Hence
//     sum_k spike_k * x_k = sum_k spike_k*hi_k + spike_k*mid_k + spike_k*lo_k
// with every product exact, accumulated in fp32 by v_mfma_f32_32x32x16_bf16:
// an fp32 contraction at three bf16 passes instead of one fp32-MFMA pass
// (bf16 MFMA runs at 16x the fp32 MFMA rate on gfx950).
//
// Used for the currents I = x W^T (x spikes, W fp32) and the weight gradient
// dW = dI^T x (dI fp32, x spikes).  Either operand may be K-contiguous or
// M/N-contiguous in memory; both are staged in LDS as [row][k] bf16 so that
// each lane's MFMA operand (8 consecutive k of one row) is one 16-byte read.
//
// Workgroup: 256 threads = 4 wave64s in 2x2, tile BM x BN x 32, wave tile
// (BM/2) x (BN/2) in 32x32 blocks.  The next k-tile is loaded into registers
// while the current one is multiplied.  Split-K as in gemm.hip.
#include <atomic>

#include "snn_internal.hpp"

namespace snn {
namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kThreads = 256;
constexpr int BK = 32;
constexpr int LDK = BK + 8;  // LDS row stride in bf16 (80 bytes)

__device__ inline uint32_t bf16_bits(float x) {
    const uint32_t b = __float_as_uint(x);
    return (b + 0x7fffu + ((b >> 16) & 1u)) >> 16;
}
__device__ inline float bf16_val(uint32_t h) { return __uint_as_float(h << 16); }

// The P bf16 parts of a value (P = 1 for spikes, which are exact).
template <int P>
__device__ inline void parts(float x, uint32_t (&h)[P]) {
    if constexpr (P == 1) {
        h[0] = bf16_bits(x);
    } else {
        h[0] = bf16_bits(x);
        const float r = x - bf16_val(h[0]);
        h[1] = bf16_bits(r);
        h[2] = bf16_bits(r - bf16_val(h[1]));
    }
}

// Raw 32-bit words of N contiguous elements of T starting at p (N*sizeof(T)
// a multiple of 4), elements past `valid` read as 0.  Vector loads of up to
// 16 bytes when the whole run is in range and aligned.
template <typename T, int N>
__device__ inline void load_words(const T *p, int valid, uint32_t (&w)[N * sizeof(T) / 4]) {
    constexpr int BYTES = N * (int)sizeof(T);
    constexpr int WORDS = BYTES / 4;
    constexpr int VB = BYTES >= 16 ? 16 : BYTES;
    if (valid >= N && (((uintptr_t)p) & (VB - 1)) == 0) {
#pragma unroll
        for (int c = 0; c < BYTES / VB; ++c) {
            const char *q = reinterpret_cast<const char *>(p) + c * VB;
            if constexpr (VB == 16) {
                const uint4 v = *reinterpret_cast<const uint4 *>(q);
                w[4 * c] = v.x; w[4 * c + 1] = v.y; w[4 * c + 2] = v.z; w[4 * c + 3] = v.w;
            } else if constexpr (VB == 8) {
                const uint2 v = *reinterpret_cast<const uint2 *>(q);
                w[2 * c] = v.x; w[2 * c + 1] = v.y;
            } else {
                w[c] = *reinterpret_cast<const uint32_t *>(q);
            }
        }
    } else {
#pragma unroll
        for (int i = 0; i < WORDS; ++i) w[i] = 0u;
#pragma unroll
        for (int i = 0; i < N; ++i) {
            if (i < valid) {
                if constexpr (sizeof(T) == 1) w[i / 4] |= (uint32_t)p[i] << (8 * (i % 4));
                else w[i] = __float_as_uint((float)p[i]);
            }
        }
    }
}

// element i of a run held as raw words
template <typename T, int WORDS>
__device__ inline float word_elem(const uint32_t (&w)[WORDS], int i) {
    if constexpr (sizeof(T) == 1) return (float)((w[i / 4] >> (8 * (i % 4))) & 0xffu);
    else return __uint_as_float(w[i]);
}

// Source formats of an operand
constexpr int SRC_SPIKE = 0;   // bytes, exact in bf16: one part
constexpr int SRC_F32 = 1;     // fp32 split into three parts while staging
constexpr int SRC_PLANES = 2;  // fp32 already split: three bf16 planes

template <int SRC>
struct SrcTraits;
template <>
struct SrcTraits<SRC_SPIKE> { typedef uint8_t T; static constexpr int P = 1, PLANES = 1; };
template <>
struct SrcTraits<SRC_F32> { typedef float T; static constexpr int P = 3, PLANES = 1; };
template <>
struct SrcTraits<SRC_PLANES> { typedef uint16_t T; static constexpr int P = 3, PLANES = 3; };

// Operand tile of R rows x BK k, P bf16 parts, into LDS [P][R][LDK].
// Each thread owns EPT = R/8 consecutive k of one row and writes them to LDS
// as 16-byte chunks of that row (row stride 80 bytes: eight consecutive rows
// cover all 32 banks, so the writes and the MFMA operand reads are free of
// bank conflicts).
//  KC (row-major [row][k]): two threads per row, each one vector load.
//  MN ([k][row]): consecutive threads take consecutive rows and gather their
//  k-run one element per k; each such load is contiguous across the wave.
// Loaded data stays packed (spike bytes four to a register) until the LDS
// store converts it; pre-split planes are copied as they are.
template <int SRC, bool KC, int R>
struct Operand {
    typedef typename SrcTraits<SRC>::T T;
    static constexpr int P = SrcTraits<SRC>::P;
    static constexpr int PL = SrcTraits<SRC>::PLANES;
    static constexpr int EPT = R * BK / kThreads;  // elements per thread
    static_assert(EPT == 8 || EPT == 16 || EPT == 32, "tile");
    static constexpr int TPR = BK / EPT;           // threads per row
    static constexpr int WORDS = EPT * (int)sizeof(T) / 4;
    uint32_t w[PL][WORDS];

    __device__ static inline int row_of(int tid) { return KC ? tid / TPR : tid % R; }
    __device__ static inline int k_of(int tid) { return KC ? (tid % TPR) * EPT : (tid / R) * EPT; }

    __device__ inline void fetch(const T *base, int64_t ld, int64_t ps, int rows, int row0, int k0,
                                 int kend) {
        const int tid = threadIdx.x;
        const int row = row0 + row_of(tid), k = k0 + k_of(tid);
        const int valid = (row < rows) ? max(0, min(EPT, kend - k)) : 0;
#pragma unroll
        for (int pl = 0; pl < PL; ++pl) {
            if constexpr (KC) {
                if (valid > 0) load_words<T, EPT>(base + pl * ps + (int64_t)row * ld + k, valid, w[pl]);
                else {
#pragma unroll
                    for (int i = 0; i < WORDS; ++i) w[pl][i] = 0u;
                }
            } else {
#pragma unroll
                for (int i = 0; i < WORDS; ++i) w[pl][i] = 0u;
                const T *col = base + pl * ps + (int64_t)k * ld + row;
#pragma unroll
                for (int j = 0; j < EPT; ++j) {
                    if (j < valid) {
                        const T e = col[(int64_t)j * ld];
                        if constexpr (sizeof(T) == 1) w[pl][j / 4] |= (uint32_t)e << (8 * (j % 4));
                        else if constexpr (sizeof(T) == 2) w[pl][j / 2] |= (uint32_t)e << (16 * (j % 2));
                        else w[pl][j] = __float_as_uint(e);
                    }
                }
            }
        }
    }

    __device__ inline void store(uint16_t *lds) const {
        const int tid = threadIdx.x;
        const int r = row_of(tid), kk = k_of(tid);
        uint32_t packed[P][EPT / 2];
        if constexpr (SRC == SRC_PLANES) {
#pragma unroll
            for (int p = 0; p < P; ++p)
#pragma unroll
                for (int i = 0; i < EPT / 2; ++i) packed[p][i] = w[p][i];
        } else {
#pragma unroll
            for (int i = 0; i < EPT; i += 2) {
                uint32_t a[P], b[P];
                parts<P>(word_elem<T, WORDS>(w[0], i), a);
                parts<P>(word_elem<T, WORDS>(w[0], i + 1), b);
#pragma unroll
                for (int p = 0; p < P; ++p) packed[p][i / 2] = a[p] | (b[p] << 16);
            }
        }
#pragma unroll
        for (int p = 0; p < P; ++p) {
            uint16_t *dst = lds + ((size_t)p * R + r) * LDK + kk;
#pragma unroll
            for (int c = 0; c < EPT / 8; ++c)
                *reinterpret_cast<uint4 *>(dst + 8 * c) = make_uint4(
                    packed[p][4 * c], packed[p][4 * c + 1], packed[p][4 * c + 2], packed[p][4 * c + 3]);
        }
    }
};

// Three bf16 planes of an fp32 array: dst[p*n + i] = part p of src[i].
__global__ __launch_bounds__(kThreads) void split_planes_kernel(const float *__restrict__ src,
                                                                uint16_t *__restrict__ dst,
                                                                int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (i >= n) return;
    uint32_t h[3];
    parts<3>(src[i], h);
    dst[i] = (uint16_t)h[0];
    dst[n + i] = (uint16_t)h[1];
    dst[2 * n + i] = (uint16_t)h[2];
}

template <int SA, bool A_KC, int SB, bool B_KC, int BM, int BN>
__global__ __launch_bounds__(kThreads, (BM * BN > 16384) ? 2 : 1) void gemm_bf16_kernel(
    int M, int N, int K, int k_chunk, int tiles_n, const typename SrcTraits<SA>::T *__restrict__ A,
    int64_t lda, int64_t a_ps, const typename SrcTraits<SB>::T *__restrict__ B, int64_t ldb,
    int64_t b_ps, float *__restrict__ C, int64_t ldc, int64_t split_stride,
    const float *__restrict__ bias) {
    constexpr int PA = SrcTraits<SA>::P, PB = SrcTraits<SB>::P;
    static_assert(PA * PB <= 3, "one operand must be exact in bf16");
    constexpr int WM = BM / 2, WN = BN / 2;
    constexpr int FM = WM / 32, FN = WN / 32;
    __shared__ __attribute__((aligned(16))) uint16_t As[PA * BM * LDK];
    __shared__ __attribute__((aligned(16))) uint16_t Bs[PB * BN * LDK];

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
    const int wm = wave & 1, wn = wave >> 1;

    floatx16 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    Operand<SA, A_KC, BM> oa;
    Operand<SB, B_KC, BN> ob;
    if (kbeg < kend) {
        oa.fetch(A, lda, a_ps, M, m0, kbeg, kend);
        ob.fetch(B, ldb, b_ps, N, n0, kbeg, kend);
    }
    const int lrow = lane & 31, lk = 8 * (lane >> 5);
    for (int k0 = kbeg; k0 < kend; k0 += BK) {
        __syncthreads();
        oa.store(As);
        ob.store(Bs);
        __syncthreads();
        if (k0 + BK < kend) {
            oa.fetch(A, lda, a_ps, M, m0, k0 + BK, kend);
            ob.fetch(B, ldb, b_ps, N, n0, k0 + BK, kend);
        }
#pragma unroll
        for (int ks = 0; ks < BK; ks += 16) {
            bf16x8 a[PA][FM], b[PB][FN];
#pragma unroll
            for (int p = 0; p < PA; ++p)
#pragma unroll
                for (int i = 0; i < FM; ++i)
                    a[p][i] = *reinterpret_cast<const bf16x8 *>(
                        As + ((size_t)p * BM + wm * WM + i * 32 + lrow) * LDK + ks + lk);
#pragma unroll
            for (int q = 0; q < PB; ++q)
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    b[q][j] = *reinterpret_cast<const bf16x8 *>(
                        Bs + ((size_t)q * BN + wn * WN + j * 32 + lrow) * LDK + ks + lk);
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j) {
                    // smallest parts first
#pragma unroll
                    for (int p = PA - 1; p >= 0; --p)
#pragma unroll
                        for (int q = PB - 1; q >= 0; --q)
                            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[p][i], b[q][j],
                                                                                acc[i][j], 0, 0, 0);
                }
        }
    }

    // 32x32 block: lane holds column (lane & 31); register r holds row
    // 8*(r/4) + 4*(lane/32) + r%4.
    float *Cz = C + (int64_t)zk * split_stride;
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            const int n = n0 + wn * WN + j * 32 + (lane & 31);
            if (n >= N) continue;
            const float bn = bias ? bias[n] : 0.f;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int m = m0 + wm * WM + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
                if (m < M) Cz[(int64_t)m * ldc + n] = acc[i][j][r] + bn;
            }
        }
}

}  // namespace

// ---- planning -------------------------------------------------------------
// Tile shapes: 0 = 128x128, 1 = 128x64, 2 = 256x128 and 3 = 128x256 (the
// long side on the spike operand).  Per MFMA a wave reads 1/F_spike +
// 1/(3 F_split) operand fragments from LDS (F = 32x32 blocks along that side
// of its wave tile), so long spike sides cut LDS traffic: 0.67 fragments per
// MFMA at 128x128, 0.42 at 256x128.
constexpr int kShapes = 4;
constexpr int kShapeBM[kShapes] = {128, 128, 256, 128};
constexpr int kShapeBN[kShapes] = {128, 64, 128, 256};
// Relative time per unit of tile work, measured on MI355X for the forward
// contraction of the 784-1000 layer (128x128 = 1).
constexpr float kShapeCost[kShapes] = {1.0f, 1.6f, 0.7f, 0.85f};
constexpr int kMaxSlotsPerCu = 8;  // upper bound on resident 256-thread blocks

struct Bf16Plan {
    int shape, BM, BN, tiles_m, tiles_n, splits, k_chunk;
    bool presplit;       // split the fp32 operand into bf16 planes once, up front
    size_t plane_bytes;  // workspace for those planes
    size_t part_bytes;   // workspace for split-K partial sums
};

static int max_splits(int tiles, int ksteps) {
    // bounded by the most blocks a device could hold and by 4 k-tiles per split
    int S = (kMaxSlotsPerCu * 256 + tiles - 1) / tiles;
    S = min(S, max(1, ksteps / 4));
    return max(1, min(S, 64));
}

static void finish_plan(Bf16Plan &p, int M, int N, int K, bool a_f32, bool f32_kc, int S) {
    const int ksteps = (K + BK - 1) / BK;
    p.k_chunk = ((ksteps + S - 1) / S) * BK;
    p.splits = (K + p.k_chunk - 1) / p.k_chunk;
    // Every workgroup along the other output side re-stages the fp32 operand;
    // when that is 16 or more times, split it once into planes instead.
    const int reuse = a_f32 ? p.tiles_n : p.tiles_m;
    const int64_t f32_elems = (int64_t)(a_f32 ? M : N) * K;
    p.presplit = f32_kc && reuse >= 16;
    p.plane_bytes = p.presplit ? align_up((size_t)3 * f32_elems * sizeof(uint16_t)) : 0;
    p.part_bytes = p.splits > 1 ? align_up((size_t)p.splits * M * N * sizeof(float)) : 0;
}

// Device-independent upper bound of the workspace any plan may use.
size_t gemm_bf16_workspace_bytes(int M, int N, int K, bool a_f32, bool f32_kc) {
    if (M < 64 || N < 64 || K <= 0) return 0;
    const int ksteps = (K + BK - 1) / BK;
    size_t best = 0;
    for (int sh = 0; sh < kShapes; ++sh) {
        Bf16Plan p{};
        p.shape = sh;
        p.BM = kShapeBM[sh];
        p.BN = kShapeBN[sh];
        p.tiles_m = (M + p.BM - 1) / p.BM;
        p.tiles_n = (N + p.BN - 1) / p.BN;
        finish_plan(p, M, N, K, a_f32, f32_kc, max_splits(p.tiles_m * p.tiles_n, ksteps));
        best = max(best, p.plane_bytes + p.part_bytes);
    }
    return best;
}

bool gemm_bf16_applies(const GemmArgs &g) {
    // exactly one spike operand and one fp32 operand, and both output sides
    // wide enough for the 128-row tiles (skinny products stay on fp32 tiles)
    if (g.M < 64 || g.N < 64) return false;
    const bool a_spk = g.a_dtype == SNN_U8, b_spk = g.b_dtype == SNN_U8;
    const bool a_f32 = g.a_dtype == SNN_F32, b_f32 = g.b_dtype == SNN_F32;
    return (a_spk && b_f32) || (a_f32 && b_spk);
}

static int device_cus() {
    static std::atomic<int> cache[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    int v = cache[dev].load(std::memory_order_relaxed);
    if (v == 0) {
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0)
            v = 256;
        cache[dev].store(v, std::memory_order_relaxed);
    }
    return v;
}

// Resident 256-thread blocks per CU of one kernel instance (runtime query,
// cached per device).
template <int SA, bool AK, int SB, bool BKc, int BM, int BN>
static int blocks_per_cu() {
    static std::atomic<int> cache[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 1;
    int v = cache[dev].load(std::memory_order_relaxed);
    if (v == 0) {
        int nb = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
                &nb, reinterpret_cast<const void *>(&gemm_bf16_kernel<SA, AK, SB, BKc, BM, BN>),
                kThreads, 0) != hipSuccess || nb <= 0)
            nb = 1;
        v = nb;
        cache[dev].store(v, std::memory_order_relaxed);
    }
    return v;
}

template <int SA, bool AK, int SB, bool BKc>
static Bf16Plan plan_for(const GemmArgs &g, bool a_f32, bool f32_kc) {
    const int cus = device_cus();
    const int ksteps = (g.K + BK - 1) / BK;
    const int occ[kShapes] = {blocks_per_cu<SA, AK, SB, BKc, 128, 128>(),
                              blocks_per_cu<SA, AK, SB, BKc, 128, 64>(),
                              blocks_per_cu<SA, AK, SB, BKc, 256, 128>(),
                              blocks_per_cu<SA, AK, SB, BKc, 128, 256>()};
    Bf16Plan best{};
    double best_cost = 1e300;
    for (int sh = 0; sh < kShapes; ++sh) {
        // the long side of shapes 2/3 goes on the spike operand
        if (sh == 2 && SA != SRC_SPIKE) continue;
        if (sh == 3 && SB != SRC_SPIKE) continue;
        Bf16Plan p{};
        p.shape = sh;
        p.BM = kShapeBM[sh];
        p.BN = kShapeBN[sh];
        p.tiles_m = (g.M + p.BM - 1) / p.BM;
        p.tiles_n = (g.N + p.BN - 1) / p.BN;
        const int tiles = p.tiles_m * p.tiles_n;
        const int slots = cus * occ[sh];
        int S = 1;
        if (tiles < slots) S = max(1, min(slots / tiles, max_splits(tiles, ksteps)));
        finish_plan(p, g.M, g.N, g.K, a_f32, f32_kc, S);
        const int64_t items = (int64_t)tiles * p.splits;
        const int64_t rounds = (items + slots - 1) / slots;
        // time ~ rounds x tile work, plus the partial-sum traffic of split-K
        double cost = (double)rounds * p.BM * p.BN * p.k_chunk * kShapeCost[sh];
        if (p.splits > 1) cost += (double)p.splits * g.M * g.N * 64.0 / cus;
        if (cost < best_cost) {
            best_cost = cost;
            best = p;
        }
    }
    return best;
}

template <int SA, bool AK, int SB, bool BKc>
static void launch_bf16_typed(const GemmArgs &g, const Bf16Plan &p, const void *A, int64_t a_ps,
                              const void *B, int64_t b_ps, float *out, int64_t ldo, int64_t ss,
                              const float *bias, hipStream_t s) {
    dim3 grid((unsigned)(p.tiles_m * p.tiles_n), 1, (unsigned)p.splits);
    const auto *a = reinterpret_cast<const typename SrcTraits<SA>::T *>(A);
    const auto *b = reinterpret_cast<const typename SrcTraits<SB>::T *>(B);
#define SNN_BF16_LAUNCH(BM_, BN_)                                                              \
    gemm_bf16_kernel<SA, AK, SB, BKc, BM_, BN_><<<grid, kThreads, 0, s>>>(                        \
        g.M, g.N, g.K, p.k_chunk, p.tiles_n, a, g.lda, a_ps, b, g.ldb, b_ps, out, ldo, ss, bias)
    switch (p.shape) {
        case 0: SNN_BF16_LAUNCH(128, 128); break;
        case 1: SNN_BF16_LAUNCH(128, 64); break;
        case 2: SNN_BF16_LAUNCH(256, 128); break;
        default: SNN_BF16_LAUNCH(128, 256); break;
    }
#undef SNN_BF16_LAUNCH
}

// Plan and launch one (source, layout) combination.
template <int SA, bool AK, int SB, bool BKc>
static hipError_t run_bf16(const GemmArgs &g, bool a_f32, void *ws, size_t ws_bytes,
                           hipStream_t s) {
    const bool f32_kc = a_f32 ? g.a_kc : g.b_kc;
    // the plan (and its presplit decision) is made for the fp32-source kernel;
    // with a presplit operand the planes kernel runs the same tile plan
    const Bf16Plan p = plan_for<SA, AK, SB, BKc>(g, a_f32, f32_kc);
    if (p.plane_bytes + p.part_bytes > 0 &&
        (ws == nullptr || ws_bytes < p.plane_bytes + p.part_bytes))
        return hipErrorInvalidValue;
    char *wsb = reinterpret_cast<char *>(ws);
    float *out = g.C;
    int64_t ldo = g.ldc, ss = 0;
    const float *bias = g.bias;
    if (p.splits > 1) {
        out = reinterpret_cast<float *>(wsb + p.plane_bytes);
        ldo = g.N;
        ss = (int64_t)g.M * g.N;
        bias = nullptr;
    }
    const void *A = g.A, *B = g.B;
    int64_t a_ps = 0, b_ps = 0;
    if (p.presplit) {
        // the fp32 operand is K-contiguous: planes keep its leading dimension
        const int rows = a_f32 ? g.M : g.N;
        const int64_t ld = a_f32 ? g.lda : g.ldb;
        const int64_t n = (int64_t)(rows - 1) * ld + g.K;
        uint16_t *planes = reinterpret_cast<uint16_t *>(wsb);
        if (p.plane_bytes < (size_t)3 * n * sizeof(uint16_t)) return hipErrorInvalidValue;
        split_planes_kernel<<<(unsigned)((n + kThreads - 1) / kThreads), kThreads, 0, s>>>(
            reinterpret_cast<const float *>(a_f32 ? g.A : g.B), planes, n);
        if constexpr (SA == SRC_F32) {
            A = planes;
            a_ps = n;
            launch_bf16_typed<SRC_PLANES, AK, SB, BKc>(g, p, A, a_ps, B, b_ps, out, ldo, ss, bias, s);
        } else {
            B = planes;
            b_ps = n;
            launch_bf16_typed<SA, AK, SRC_PLANES, BKc>(g, p, A, a_ps, B, b_ps, out, ldo, ss, bias, s);
        }
    } else {
        launch_bf16_typed<SA, AK, SB, BKc>(g, p, A, a_ps, B, b_ps, out, ldo, ss, bias, s);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (p.splits > 1) e = launch_splitk_reduce(g.M, g.N, p.splits, out, g.C, g.ldc, g.bias, s);
    return e;
}

hipError_t launch_gemm_bf16(const GemmArgs &g, void *ws, size_t ws_bytes, hipStream_t s) {
    const bool a_f32 = g.a_dtype == SNN_F32;
    if (a_f32) {
        if (g.a_kc) {
            if (g.b_kc) return run_bf16<SRC_F32, true, SRC_SPIKE, true>(g, true, ws, ws_bytes, s);
            return run_bf16<SRC_F32, true, SRC_SPIKE, false>(g, true, ws, ws_bytes, s);
        }
        if (g.b_kc) return run_bf16<SRC_F32, false, SRC_SPIKE, true>(g, true, ws, ws_bytes, s);
        return run_bf16<SRC_F32, false, SRC_SPIKE, false>(g, true, ws, ws_bytes, s);
    }
    if (g.a_kc) {
        if (g.b_kc) return run_bf16<SRC_SPIKE, true, SRC_F32, true>(g, false, ws, ws_bytes, s);
        return run_bf16<SRC_SPIKE, true, SRC_F32, false>(g, false, ws, ws_bytes, s);
    }
    if (g.b_kc) return run_bf16<SRC_SPIKE, false, SRC_F32, true>(g, false, ws, ws_bytes, s);
    return run_bf16<SRC_SPIKE, false, SRC_F32, false>(g, false, ws, ws_bytes, s);
}

}  // namespace snn
