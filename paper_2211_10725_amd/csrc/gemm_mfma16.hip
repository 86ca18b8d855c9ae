// Contractions on the 16-bit matrix cores of gfx950 with exact products.
//
//   C[M,N] = sum_k A(m,k) B(n,k) (+ bias[n]),  fp32 accumulate
//
// Operands are staged in LDS as 16-bit parts, and every product of parts is
// exact, so the result is the exactly-multiplied sum with fp32 accumulation:
//  * a spike (a byte, 0/1) is exact in bf16 and in fp16: one part;
//  * an fp32 value x splits exactly into three bf16 parts, x = hi + mid + lo:
//    hi = bf16(x) (nearest even), mid = bf16(x - hi), lo = x - hi - mid; each
//    subtraction is exact (Sterbenz), x - hi has at most 16 significant bits
//    and x - hi - mid at most 8, so lo is exact in bf16 down to the bottom of
//    the fp32 normal range;
//  * an fp16 value is exact in fp16 (one part) or in two bf16 parts (11
//    significand bits = 8 + 3, same reasoning);
//  * a bf16 value is one bf16 part.
// A contraction of parts P_A x P_B runs P_A * P_B MFMA passes (<= 6).  The
// MFMA type is fp16 when both operands are spikes or fp16 (one pass for the
// fp16 network's currents), otherwise bf16, whose exponent range holds the
// small gradients of BPTT.  bf16/fp16 MFMA run at 16x the fp32 MFMA rate.
//
// Tiles: 256 threads = 4 wave64s in 2x2, BM x BN x 32; each wave computes
// (BM/2) x (BN/2) with v_mfma_f32_32x32x16_{bf16,f16}.  Both operand layouts
// (K- or M/N-contiguous in memory) are staged as [part][row][k] with an
// 80-byte row stride, so an operand fetch (8 consecutive k of one row, 16
// bytes) and the 16-byte staging writes are free of bank conflicts.  The next
// k-tile is fetched into registers while the current one is multiplied.  Tile
// shape and split-K come from the runtime occupancy; workgroups are
// renumbered so each XCD covers a contiguous range of tiles.
#include <atomic>
#include <type_traits>

#include "snn_internal.hpp"

namespace snn {
namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 half8 __attribute__((ext_vector_type(8)));

constexpr int kThreads = 256;
constexpr int BK = 32;  // k-tile of the planning model (the kernels use 32 or 64)

constexpr int MT_BF16 = 0;
constexpr int MT_F16 = 1;

__device__ inline uint32_t bf16_bits(float x) {
    const uint32_t b = __float_as_uint(x);
    return (b + 0x7fffu + ((b >> 16) & 1u)) >> 16;
}
__device__ inline float bf16_val(uint32_t h) { return __uint_as_float(h << 16); }
__device__ inline uint32_t f16_bits(float x) {
    const _Float16 h = (_Float16)x;
    return __builtin_bit_cast(uint16_t, h);
}
__device__ inline float f16_val(uint32_t h) {
    return (float)__builtin_bit_cast(_Float16, (uint16_t)h);
}

// Source formats of an operand
constexpr int SRC_SPIKE = 0;   // bytes: one part in either MFMA type
constexpr int SRC_F32 = 1;     // fp32: three bf16 parts, split while staging
constexpr int SRC_PLANES = 2;  // fp32 already split into three bf16 planes
constexpr int SRC_H16 = 3;     // 16-bit values of the MFMA type: one part
constexpr int SRC_F16X2 = 4;   // fp16 values as two bf16 parts

template <int SRC>
struct SrcTraits;
template <>
struct SrcTraits<SRC_SPIKE> { typedef uint8_t T; static constexpr int P = 1, PLANES = 1; };
template <>
struct SrcTraits<SRC_F32> { typedef float T; static constexpr int P = 3, PLANES = 1; };
template <>
struct SrcTraits<SRC_PLANES> { typedef uint16_t T; static constexpr int P = 3, PLANES = 3; };
template <>
struct SrcTraits<SRC_H16> { typedef uint16_t T; static constexpr int P = 1, PLANES = 1; };
template <>
struct SrcTraits<SRC_F16X2> { typedef uint16_t T; static constexpr int P = 2, PLANES = 1; };

// Raw 32-bit words of N contiguous elements of T starting at p, elements past
// `valid` read as 0.  Vector loads of up to 16 bytes when the whole run is in
// range and aligned.
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
                else if constexpr (sizeof(T) == 2) w[i / 2] |= (uint32_t)p[i] << (16 * (i % 2));
                else w[i] = __float_as_uint((float)p[i]);
            }
        }
    }
}

// The 16-bit part `part` of element i (of a run held as raw words).
template <int SRC, int MT, int WORDS>
__device__ inline uint32_t part_of(const uint32_t (&w)[WORDS], int i, int part) {
    if constexpr (SRC == SRC_SPIKE) {
        // a byte has at most 8 significant bits: its fp32 value's upper half
        // is its bf16 value, no rounding needed
        const float v = (float)((w[i / 4] >> (8 * (i % 4))) & 0xffu);
        return MT == MT_F16 ? f16_bits(v) : (__float_as_uint(v) >> 16);
    } else if constexpr (SRC == SRC_H16 || SRC == SRC_PLANES) {
        return (w[i / 2] >> (16 * (i % 2))) & 0xffffu;
    } else if constexpr (SRC == SRC_F16X2) {
        const float v = f16_val((w[i / 2] >> (16 * (i % 2))) & 0xffffu);
        const uint32_t hi = bf16_bits(v);
        return part == 0 ? hi : bf16_bits(v - bf16_val(hi));
    } else {  // SRC_F32
        const float x = __uint_as_float(w[i]);
        const uint32_t hi = bf16_bits(x);
        if (part == 0) return hi;
        const float r = x - bf16_val(hi);
        const uint32_t mid = bf16_bits(r);
        if (part == 1) return mid;
        return bf16_bits(r - bf16_val(mid));
    }
}

// Operand tile of R rows x BK k, P 16-bit parts, into LDS [P][R][LDK].  Each
// thread owns EPT = R/8 consecutive k of one row and writes them as 16-byte
// chunks (eight consecutive rows cover all 32 banks).
//  KC (row-major [row][k]): two to four threads per row, one vector load each.
//  MN ([k][row]): consecutive threads take consecutive rows and gather their
//  k-run one element per k; each such load is contiguous across the wave.
template <int SRC, int MT, bool KC, int R, int BK>
struct Operand {
    typedef typename SrcTraits<SRC>::T T;
    static constexpr int P = SrcTraits<SRC>::P;
    static constexpr int PL = SrcTraits<SRC>::PLANES;
    static constexpr int LDK = BK + 8;             // LDS row stride (16-bit elements)
    static constexpr int STAGE = P * R * LDK;      // 16-bit units per LDS stage
    static constexpr int EPT = R * BK / kThreads;  // elements per thread
    static_assert(EPT == 8 || EPT == 16 || EPT == 32 || EPT == 64, "tile");
    static constexpr int TPR = BK / EPT;           // threads per row (KC)
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
#pragma unroll
        for (int p = 0; p < P; ++p) {
            uint32_t packed[EPT / 2];
            if constexpr (SRC == SRC_PLANES) {
#pragma unroll
                for (int i = 0; i < EPT / 2; ++i) packed[i] = w[p][i];
            } else if constexpr (SRC == SRC_H16) {
#pragma unroll
                for (int i = 0; i < EPT / 2; ++i) packed[i] = w[0][i];
            } else {
#pragma unroll
                for (int i = 0; i < EPT; i += 2)
                    packed[i / 2] = part_of<SRC, MT, WORDS>(w[0], i, p) |
                                    (part_of<SRC, MT, WORDS>(w[0], i + 1, p) << 16);
            }
            uint16_t *dst = lds + ((size_t)p * R + r) * LDK + kk;
#pragma unroll
            for (int c = 0; c < EPT / 8; ++c)
                *reinterpret_cast<uint4 *>(dst + 8 * c) =
                    make_uint4(packed[4 * c], packed[4 * c + 1], packed[4 * c + 2], packed[4 * c + 3]);
        }
    }
};

// Three bf16 planes of an fp32 matrix src[rows][ld] (K columns used) into
// dst[p][rows][ldp], ldp = K rounded up to 8 so that every plane row starts on
// 16 bytes; the padding columns are 0.
__global__ __launch_bounds__(kThreads) void split_planes_kernel(const float *__restrict__ src,
                                                                int64_t ld, int K, int ldp,
                                                                int64_t n,
                                                                uint16_t *__restrict__ dst) {
    const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (i >= n) return;
    const int64_t r = i / ldp;
    const int k = (int)(i - r * ldp);
    uint32_t w[1] = {k < K ? __float_as_uint(src[r * ld + k]) : 0u};
    dst[i] = (uint16_t)part_of<SRC_F32, MT_BF16, 1>(w, 0, 0);
    dst[n + i] = (uint16_t)part_of<SRC_F32, MT_BF16, 1>(w, 0, 1);
    dst[2 * n + i] = (uint16_t)part_of<SRC_F32, MT_BF16, 1>(w, 0, 2);
}

// Operand tile stored M/N-contiguous ([k][row], the layout of dL/dI and of
// the spikes x in the weight gradient dW = dI^T x) without a transpose in
// global memory.  The tile is copied in its own layout into LDS with
// coalesced 16-byte loads along the rows ([part][k][row], rows of RS 16-bit
// elements or RSB bytes), and the MFMA fragments are read with gfx950's
// transposing LDS loads: within each 16 lanes, ds_read_b64_tr_b16 hands lane
// i element e of lane 4e + i/4's 4-element run (position i % 4), and
// ds_read_b64_tr_b8 element e of lane 2e + i/8's 8-byte run (position i % 8)
// (measured on the GPU with an in-bounds probe).  With lane L of a group
// pointing at k-row kb + L/4 (16-bit) or kb + L/2 (bytes) and row j0 +
// 4 (L % 4) or j0 + 8 (L % 2), lane i receives k = kb, kb+1, ... of row j0 + i:
// the k-contiguous run the MFMA operand needs.  fp32 is split into its three
// exact bf16 parts while staged.  Row strides put the 4 (or 8) k-rows a group
// reads on distinct banks: RS = 16 mod 64 elements, RSB = 16 mod 128 bytes.
typedef short v4s16 __attribute__((ext_vector_type(4)));
typedef int v2i32 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) v4s16 lds_v4s16;
typedef __attribute__((address_space(3))) v2i32 lds_v2i32;

template <int SRC>
constexpr bool mn_staged() {
    return SRC == SRC_SPIKE || SRC == SRC_H16 || SRC == SRC_PLANES || SRC == SRC_F32;
}

template <int SRC, int MT, int R, int BK>
struct OperandMN {
    typedef typename SrcTraits<SRC>::T T;
    static constexpr int P = SrcTraits<SRC>::P;
    static constexpr int PL = SrcTraits<SRC>::PLANES;
    static constexpr bool BYTES = SRC == SRC_SPIKE;
    static constexpr int RS = (R + 63) / 64 * 64 + 16;    // 16-bit elements per k-row
    static constexpr int RSB = (R + 127) / 128 * 128 + 16; // bytes per k-row (spikes)
    static constexpr int STAGE = BYTES ? BK * RSB / 2 : P * BK * RS;  // 16-bit units
    static constexpr int VE = 16 / (int)sizeof(T);         // elements per 16-byte run
    static constexpr int CPR = R / VE;                     // runs per k-row
    static constexpr int RUNS = BK * CPR;                  // runs per tile (per plane)
    static constexpr int CPT = (RUNS + kThreads - 1) / kThreads;  // runs per thread
    uint4 v[PL][CPT];

    __device__ inline void fetch(const T *base, int64_t ld, int64_t ps, int rows, int row0, int k0,
                                 int kend) {
        const bool vec = ((((uintptr_t)base) | (uintptr_t)(ld * (int64_t)sizeof(T)) |
                           (uintptr_t)(ps * (int64_t)sizeof(T))) & 15) == 0;
#pragma unroll
        for (int c = 0; c < CPT; ++c) {
            const int q = threadIdx.x + c * kThreads;
            const int kr = q / CPR, row = row0 + (q % CPR) * VE, k = k0 + kr;
            const int valid = (q < RUNS && k < kend) ? min(VE, rows - row) : 0;
#pragma unroll
            for (int pl = 0; pl < PL; ++pl) {
                const T *src = base + pl * ps + (int64_t)k * ld + row;
                if (valid == VE && vec) {
                    v[pl][c] = *reinterpret_cast<const uint4 *>(src);
                } else {
                    uint32_t w[4] = {0u, 0u, 0u, 0u};
#pragma unroll
                    for (int e = 0; e < VE; ++e) {
                        if (e < valid) {
                            if constexpr (sizeof(T) == 1) w[e / 4] |= (uint32_t)src[e] << (8 * (e % 4));
                            else if constexpr (sizeof(T) == 2) w[e / 2] |= (uint32_t)src[e] << (16 * (e % 2));
                            else w[e] = __float_as_uint(src[e]);
                        }
                    }
                    v[pl][c] = make_uint4(w[0], w[1], w[2], w[3]);
                }
            }
        }
    }

    __device__ inline void store(uint16_t *lds) const {
#pragma unroll
        for (int c = 0; c < CPT; ++c) {
            const int q = threadIdx.x + c * kThreads;
            if (RUNS % kThreads != 0 && q >= RUNS) break;
            const int kr = q / CPR, col = (q % CPR) * VE;
            if constexpr (BYTES) {
                *reinterpret_cast<uint4 *>(reinterpret_cast<uint8_t *>(lds) + kr * RSB + col) = v[0][c];
            } else if constexpr (SRC == SRC_F32) {
                // four fp32 values -> their hi, mid, lo bf16 parts
                const uint32_t x[4] = {v[0][c].x, v[0][c].y, v[0][c].z, v[0][c].w};
                uint32_t hp[3][4];
#pragma unroll
                for (int e = 0; e < 4; ++e)
#pragma unroll
                    for (int p = 0; p < 3; ++p) hp[p][e] = part_of<SRC_F32, MT, 4>(x, e, p);
#pragma unroll
                for (int p = 0; p < 3; ++p)
                    *reinterpret_cast<uint2 *>(lds + (p * BK + kr) * RS + col) =
                        make_uint2(hp[p][0] | (hp[p][1] << 16), hp[p][2] | (hp[p][3] << 16));
            } else {
#pragma unroll
                for (int p = 0; p < P; ++p)
                    *reinterpret_cast<uint4 *>(lds + (p * BK + kr) * RS + col) = v[p][c];
            }
        }
    }

    // the MFMA fragment of part p for operand rows r0 .. r0 + 31 and k-step ks
    __device__ static inline uint4 frag(const uint16_t *lds, int p, int r0, int ks, int lane) {
        const int g = lane >> 4, L = lane & 15;
        const int j0 = r0 + 16 * (g & 1), kb = ks + 8 * (g >> 1);
        if constexpr (BYTES) {
            const uint8_t *b = reinterpret_cast<const uint8_t *>(lds) + (kb + (L >> 1)) * RSB + j0 + 8 * (L & 1);
            const v2i32 r = __builtin_amdgcn_ds_read_tr8_b64_v2i32((lds_v2i32 *)b);
            uint2 raw;
            raw.x = (uint32_t)r[0];
            raw.y = (uint32_t)r[1];
            uint32_t o[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const uint32_t wd = i < 2 ? raw.x : raw.y;
                const float lo = (float)((wd >> (16 * (i % 2))) & 0xffu);
                const float hi = (float)((wd >> (16 * (i % 2) + 8)) & 0xffu);
                if constexpr (MT == MT_F16)
                    o[i] = f16_bits(lo) | (f16_bits(hi) << 16);
                else
                    o[i] = (__float_as_uint(lo) >> 16) | (__float_as_uint(hi) & 0xffff0000u);
            }
            return make_uint4(o[0], o[1], o[2], o[3]);
        } else {
            const uint16_t *a = lds + (p * BK + kb + (L >> 2)) * RS + j0 + 4 * (L & 3);
            const v4s16 r0v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s16 *)a);
            const v4s16 r1v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s16 *)(a + 4 * RS));
            const uint2 x0 = __builtin_bit_cast(uint2, r0v), x1 = __builtin_bit_cast(uint2, r1v);
            return make_uint4(x0.x, x0.y, x1.x, x1.y);
        }
    }
};

template <int MT>
__device__ inline floatx16 mfma32(const uint4 &a, const uint4 &b, const floatx16 &c) {
    if constexpr (MT == MT_F16)
        return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(half8, a),
                                                      __builtin_bit_cast(half8, b), c, 0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                       __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// k-tile and LDS stages: single-part operand pairs use 64-deep k-tiles in a
// two-stage LDS ring (one barrier per k-tile, the next tile staged while this
// one is multiplied); multi-part pairs carry P times the MFMA work per staged
// byte and use 32-deep k-tiles, in two stages too when they have at most three
// parts and the A side is not spikes (the weight gradient dI x, the fp16
// net's input gradient: measured faster), else in a single stage (two
// barriers), which leaves LDS for more resident workgroups (the forward
// spikes x W: measured faster).
template <int SA, int SB>
constexpr int ktile() { return SrcTraits<SA>::P * SrcTraits<SB>::P == 1 ? 64 : 32; }
template <int SA, int SB>
constexpr int lds_stages() {
    constexpr int parts = SrcTraits<SA>::P * SrcTraits<SB>::P;
    return (parts == 1 || (parts <= 3 && SA != SRC_SPIKE)) ? 2 : 1;
}

template <int MT, int SA, bool A_KC, int SB, bool B_KC, int BM, int BN, bool POOL = false>
__global__ __launch_bounds__(kThreads, (BM * BN > 16384) ? 2 : 1) void gemm16_kernel(
    int M, int N, int K, int k_chunk, int tiles_n, const typename SrcTraits<SA>::T *__restrict__ A,
    int64_t lda, int64_t a_ps, const typename SrcTraits<SB>::T *__restrict__ B, int64_t ldb,
    int64_t b_ps, float *__restrict__ C, int64_t ldc, int64_t split_stride,
    const float *__restrict__ bias, int pool_hw, float *__restrict__ pool_cur,
    uint8_t *__restrict__ pool_arg) {
    constexpr int PA = SrcTraits<SA>::P, PB = SrcTraits<SB>::P;
    static_assert(PA * PB <= 6, "at most six passes");
    constexpr int KT = ktile<SA, SB>();
    constexpr int LDK = KT + 8;
    constexpr int WM = BM / 2, WN = BN / 2;
    constexpr int FM = WM / 32, FN = WN / 32;
    using OA = std::conditional_t<!A_KC && mn_staged<SA>(), OperandMN<SA, MT, BM, KT>,
                                  Operand<SA, MT, A_KC, BM, KT>>;
    using OB = std::conditional_t<!B_KC && mn_staged<SB>(), OperandMN<SB, MT, BN, KT>,
                                  Operand<SB, MT, B_KC, BN, KT>>;
    constexpr bool A_MN = !A_KC && mn_staged<SA>(), B_MN = !B_KC && mn_staged<SB>();
    constexpr int SZA = OA::STAGE, SZB = OB::STAGE;
    constexpr int NS = lds_stages<SA, SB>();
    __shared__ __attribute__((aligned(16))) uint16_t As[NS * SZA];
    __shared__ __attribute__((aligned(16))) uint16_t Bs[NS * SZB];

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

    OA oa;
    OB ob;
    // prologue: stage the first k-tile (two-stage ring) and fetch the next
    if (kbeg < kend) {
        oa.fetch(A, lda, a_ps, M, m0, kbeg, kend);
        ob.fetch(B, ldb, b_ps, N, n0, kbeg, kend);
        if constexpr (NS == 2) {
            oa.store(As);
            ob.store(Bs);
            if (kbeg + KT < kend) {
                oa.fetch(A, lda, a_ps, M, m0, kbeg + KT, kend);
                ob.fetch(B, ldb, b_ps, N, n0, kbeg + KT, kend);
            }
        }
    }
    if constexpr (NS == 2) __syncthreads();
    const int lrow = lane & 31, lk = 8 * (lane >> 5);
    int stage = 0;
    for (int k0 = kbeg; k0 < kend; k0 += KT) {
        if constexpr (NS == 1) {
            // single stage: stage this tile, then fetch the next while multiplying
            __syncthreads();
            oa.store(As);
            ob.store(Bs);
            __syncthreads();
            if (k0 + KT < kend) {
                oa.fetch(A, lda, a_ps, M, m0, k0 + KT, kend);
                ob.fetch(B, ldb, b_ps, N, n0, k0 + KT, kend);
            }
        }
        const uint16_t *as = As + stage * SZA;
        const uint16_t *bs = Bs + stage * SZB;
#pragma unroll
        for (int ks = 0; ks < KT; ks += 16) {
            uint4 a[PA][FM], b[PB][FN];
#pragma unroll
            for (int p = 0; p < PA; ++p)
#pragma unroll
                for (int i = 0; i < FM; ++i) {
                    if constexpr (A_MN)
                        a[p][i] = OA::frag(as, p, wm * WM + i * 32, ks, lane);
                    else
                        a[p][i] = *reinterpret_cast<const uint4 *>(
                            as + ((size_t)p * BM + wm * WM + i * 32 + lrow) * LDK + ks + lk);
                }
#pragma unroll
            for (int q = 0; q < PB; ++q)
#pragma unroll
                for (int j = 0; j < FN; ++j) {
                    if constexpr (B_MN)
                        b[q][j] = OB::frag(bs, q, wn * WN + j * 32, ks, lane);
                    else
                        b[q][j] = *reinterpret_cast<const uint4 *>(
                            bs + ((size_t)q * BN + wn * WN + j * 32 + lrow) * LDK + ks + lk);
                }
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j) {
                    // smallest parts first
#pragma unroll
                    for (int p = PA - 1; p >= 0; --p)
#pragma unroll
                        for (int q = PB - 1; q >= 0; --q)
                            acc[i][j] = mfma32<MT>(a[p][i], b[q][j], acc[i][j]);
                }
        }
        if constexpr (NS == 2) {
            // stage the next k-tile into the other buffer (last read before the
            // previous barrier), then fetch the one after it
            if (k0 + KT < kend) {
                oa.store(As + (stage ^ 1) * SZA);
                ob.store(Bs + (stage ^ 1) * SZB);
                if (k0 + 2 * KT < kend) {
                    oa.fetch(A, lda, a_ps, M, m0, k0 + 2 * KT, kend);
                    ob.fetch(B, ldb, b_ps, N, n0, k0 + 2 * KT, kend);
                }
            }
            __syncthreads();
            stage ^= 1;
        }
    }

    // 32x32 block: lane holds column (lane & 31); register r holds row
    // 8*(r/4) + 4*(lane/32) + r%4.
    if constexpr (POOL) {
        // registers 4g .. 4g + 3 of a lane are the four rows of one pool
        // window (M is a multiple of 4): the first maximum of C + bias
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j) {
                const int n = n0 + wn * WN + j * 32 + (lane & 31);
                if (n >= N) continue;
                const float bn = bias ? bias[n] : 0.f;
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const int m = m0 + wm * WM + i * 32 + 8 * g + 4 * (lane >> 5);
                    if (m >= M) continue;
                    float best = acc[i][j][4 * g] + bn;
                    int a = 0;
#pragma unroll
                    for (int d = 1; d < 4; ++d) {
                        const float v = acc[i][j][4 * g + d] + bn;
                        if (v > best) {
                            best = v;
                            a = d;
                        }
                    }
                    const int q = m >> 2, nb = q / pool_hw;
                    const int64_t o = ((int64_t)nb * N + n) * pool_hw + (q - nb * pool_hw);
                    pool_cur[o] = best;
                    pool_arg[o] = (uint8_t)a;
                }
            }
        return;
    }
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

// ---- planning -------------------------------------------------------------
// Tile shapes: 0 = 128x128, 1 = 128x64, 2 = 256x128 (long side on A) and
// 3 = 128x256 (long side on B).  Per MFMA a wave reads 1/F_a' + 1/F_b'
// fragments (F' = 32x32 blocks on that side of its wave tile divided by the
// other side's part count), so the long side goes on the operand with fewer
// parts.
constexpr int kShapes = 4;
constexpr int kShapeBM[kShapes] = {128, 128, 256, 128};
constexpr int kShapeBN[kShapes] = {128, 64, 128, 256};
// Relative time per unit of tile work (128x128 = 1), measured on MI355X with
// every shape forced in turn on the contractions of the dense benchmark
// layers: [multi-part kernels, single-part kernels][shape].
constexpr float kShapeCost[2][kShapes] = {{1.0f, 1.6f, 0.6f, 0.85f}, {1.0f, 1.3f, 1.2f, 1.2f}};
constexpr int kMaxSlotsPerCu = 8;  // upper bound on resident 256-thread blocks

struct Plan16 {
    int shape, BM, BN, tiles_m, tiles_n, splits, k_chunk;
    bool presplit;       // split the fp32 operand into bf16 planes once, up front
    size_t plane_bytes;  // workspace for those planes
    size_t part_bytes;   // workspace for split-K partial sums
};

int max_splits(int tiles, int ksteps, int64_t mn) {
    // bounded by the most blocks a device could hold and by 4 k-tiles per
    // split; a small output over a long K (a conv weight gradient) may split
    // further, its partial sums staying small
    int S = (kMaxSlotsPerCu * 256 + tiles - 1) / tiles;
    S = min(S, max(1, ksteps / 4));
    return max(1, min(S, mn <= 65536 ? 256 : 64));
}

// Operand classification --------------------------------------------------
struct Kind {
    int mt;        // MFMA type
    int sa, sb;    // source formats
    bool ok;       // a supported combination
};

int parts_of(int src) {
    switch (src) {
        case SRC_F32: case SRC_PLANES: return 3;
        case SRC_F16X2: return 2;
        default: return 1;
    }
}

Kind classify(int a_dtype, int b_dtype) {
    Kind k{};
    auto f16ish = [](int t) { return t == SNN_U8 || t == SNN_F16; };
    k.mt = (f16ish(a_dtype) && f16ish(b_dtype)) ? MT_F16 : MT_BF16;
    auto src = [&](int t, bool &ok) {
        switch (t) {
            case SNN_U8: return SRC_SPIKE;
            case SNN_F32: return SRC_F32;
            case SNN_BF16: return SRC_H16;
            case kPlanes3: return SRC_PLANES;
            case SNN_F16: return k.mt == MT_F16 ? SRC_H16 : SRC_F16X2;
            default: ok = false; return SRC_SPIKE;
        }
    };
    bool ok = true;
    k.sa = src(a_dtype, ok);
    k.sb = src(b_dtype, ok);
    k.ok = ok && parts_of(k.sa) * parts_of(k.sb) <= 6;
    return k;
}

void finish_plan(Plan16 &p, int M, int N, int K, const Kind &kd, bool a_kc, bool b_kc, int S) {
    // split boundaries on whole k-tiles of the kernel that will run
    const int kt = parts_of(kd.sa) * parts_of(kd.sb) == 1 ? 64 : 32;
    const int ksteps = (K + kt - 1) / kt;
    p.k_chunk = ((ksteps + S - 1) / S) * kt;
    p.splits = (K + p.k_chunk - 1) / p.k_chunk;
    // An fp32 operand against spikes is re-staged by every workgroup along the
    // other output side; when that is 16 or more times, split it once into
    // planes instead.
    p.presplit = false;
    int64_t f32_elems = 0;
    const int64_t ldp = (K + 7) / 8 * 8;  // plane rows padded to 16 bytes
    if (kd.sa == SRC_F32 && kd.sb == SRC_SPIKE && a_kc) {
        p.presplit = p.tiles_n >= 16;
        f32_elems = (int64_t)M * ldp;
    } else if (kd.sb == SRC_F32 && kd.sa == SRC_SPIKE && b_kc) {
        p.presplit = p.tiles_m >= 16;
        f32_elems = (int64_t)N * ldp;
    }
    p.plane_bytes = p.presplit ? align_up((size_t)3 * f32_elems * sizeof(uint16_t)) : 0;
    p.part_bytes = p.splits > 1 ? align_up((size_t)p.splits * M * N * sizeof(float)) : 0;
}

bool shape_allowed(int sh, const Kind &kd) {
    if (sh == 2) return parts_of(kd.sa) <= parts_of(kd.sb);
    if (sh == 3) return parts_of(kd.sb) <= parts_of(kd.sa);
    return true;
}

// Resident 256-thread blocks per CU of one kernel instance (runtime query,
// cached per device).
template <int MT, int SA, bool AK, int SB, bool BKc, int BM, int BN>
int blocks_per_cu() {
    static std::atomic<int> cache[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 1;
    int v = cache[dev].load(std::memory_order_relaxed);
    if (v == 0) {
        int nb = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
                &nb, reinterpret_cast<const void *>(&gemm16_kernel<MT, SA, AK, SB, BKc, BM, BN>),
                kThreads, 0) != hipSuccess || nb <= 0)
            nb = 1;
        v = nb;
        cache[dev].store(v, std::memory_order_relaxed);
    }
    return v;
}

template <int MT, int SA, bool AK, int SB, bool BKc>
Plan16 plan_for(const GemmArgs &g, const Kind &kd) {
    const int cus = device_cus();
    const int ksteps = (g.K + BK - 1) / BK;
    const int occ[kShapes] = {blocks_per_cu<MT, SA, AK, SB, BKc, 128, 128>(),
                              blocks_per_cu<MT, SA, AK, SB, BKc, 128, 64>(),
                              blocks_per_cu<MT, SA, AK, SB, BKc, 256, 128>(),
                              blocks_per_cu<MT, SA, AK, SB, BKc, 128, 256>()};
    Plan16 best{};
    double best_cost = 1e300;
    for (int sh = 0; sh < kShapes; ++sh) {
        if (!shape_allowed(sh, kd)) continue;
        Plan16 p{};
        p.shape = sh;
        p.BM = kShapeBM[sh];
        p.BN = kShapeBN[sh];
        p.tiles_m = (g.M + p.BM - 1) / p.BM;
        p.tiles_n = (g.N + p.BN - 1) / p.BN;
        const int tiles = p.tiles_m * p.tiles_n;
        const int slots = cus * occ[sh];
        int S = 1;
        if (tiles < slots) S = max(1, min(slots / tiles, max_splits(tiles, ksteps, (int64_t)g.M * g.N)));
        finish_plan(p, g.M, g.N, g.K, kd, g.a_kc, g.b_kc, S);
        const int64_t items = (int64_t)tiles * p.splits;
        const int64_t rounds = (items + slots - 1) / slots;
        // time ~ rounds x tile work, plus the partial-sum traffic of split-K
        double cost = (double)rounds * p.BM * p.BN * p.k_chunk *
                      kShapeCost[SrcTraits<SA>::P * SrcTraits<SB>::P == 1 ? 1 : 0][sh];
        if (p.splits > 1) cost += (double)p.splits * g.M * g.N * 64.0 / cus;
        if (cost < best_cost) {
            best_cost = cost;
            best = p;
        }
    }
    return best;
}

template <int MT, int SA, bool AK, int SB, bool BKc, bool POOL = false>
void launch16(const GemmArgs &g, const Plan16 &p, const void *A, int64_t a_ps, const void *B,
              int64_t b_ps, float *out, int64_t ldo, int64_t ss, const float *bias, hipStream_t s) {
    dim3 grid((unsigned)(p.tiles_m * p.tiles_n), 1, (unsigned)p.splits);
    const auto *a = reinterpret_cast<const typename SrcTraits<SA>::T *>(A);
    const auto *b = reinterpret_cast<const typename SrcTraits<SB>::T *>(B);
#define SNN_G16_LAUNCH(BM_, BN_)                                                                \
    gemm16_kernel<MT, SA, AK, SB, BKc, BM_, BN_, POOL><<<grid, kThreads, 0, s>>>(                  \
        g.M, g.N, g.K, p.k_chunk, p.tiles_n, a, g.lda, a_ps, b, g.ldb, b_ps, out, ldo, ss, bias,   \
        g.pool_hw, g.pool_cur, g.pool_arg)
    switch (p.shape) {
        case 0: SNN_G16_LAUNCH(128, 128); break;
        case 1: SNN_G16_LAUNCH(128, 64); break;
        case 2: SNN_G16_LAUNCH(256, 128); break;
        default: SNN_G16_LAUNCH(128, 256); break;
    }
#undef SNN_G16_LAUNCH
}

// Plan and launch one (type, sources, layouts) combination.
template <int MT, int SA, bool AK, int SB, bool BKc>
hipError_t run16(const GemmArgs &g, const Kind &kd, void *ws, size_t ws_bytes, hipStream_t s) {
    const Plan16 p = plan_for<MT, SA, AK, SB, BKc>(g, kd);
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
    // the pool epilogue: spikes against fp32 weights (a convolution's
    // forward), one pass over K, whole windows
    constexpr bool CAN_POOL = MT == MT_BF16 && SA == SRC_SPIKE && SB == SRC_F32 && AK && BKc;
    const bool pool = g.pool_hw > 0 && g.pooled && p.splits == 1 && g.M % 4 == 0;
    if constexpr ((SA == SRC_F32 && SB == SRC_SPIKE) || (SB == SRC_F32 && SA == SRC_SPIKE)) {
        if (p.presplit) {
            // the fp32 operand is K-contiguous; its planes get 16-byte rows
            constexpr bool a_f32 = SA == SRC_F32;
            const int rows = a_f32 ? g.M : g.N;
            const int ldp = (g.K + 7) / 8 * 8;
            const int64_t n = (int64_t)rows * ldp;
            uint16_t *planes = reinterpret_cast<uint16_t *>(wsb);
            if (p.plane_bytes < (size_t)3 * n * sizeof(uint16_t)) return hipErrorInvalidValue;
            split_planes_kernel<<<(unsigned)((n + kThreads - 1) / kThreads), kThreads, 0, s>>>(
                reinterpret_cast<const float *>(a_f32 ? g.A : g.B), a_f32 ? g.lda : g.ldb, g.K,
                ldp, n, planes);
            GemmArgs gp = g;
            if constexpr (a_f32) {
                gp.lda = ldp;
                launch16<MT, SRC_PLANES, AK, SB, BKc>(gp, p, planes, n, g.B, 0, out, ldo, ss, bias, s);
            } else {
                gp.ldb = ldp;
                if constexpr (CAN_POOL) {
                    if (pool) {
                        launch16<MT, SA, AK, SRC_PLANES, BKc, true>(gp, p, g.A, 0, planes, n, out,
                                                                    ldo, ss, bias, s);
                        *g.pooled = true;
                    } else {
                        launch16<MT, SA, AK, SRC_PLANES, BKc>(gp, p, g.A, 0, planes, n, out, ldo,
                                                              ss, bias, s);
                    }
                } else {
                    launch16<MT, SA, AK, SRC_PLANES, BKc>(gp, p, g.A, 0, planes, n, out, ldo, ss,
                                                          bias, s);
                }
            }
        } else if constexpr (CAN_POOL) {
            if (pool) {
                launch16<MT, SA, AK, SB, BKc, true>(g, p, g.A, g.a_ps, g.B, g.b_ps, out, ldo, ss,
                                                    bias, s);
                *g.pooled = true;
            } else {
                launch16<MT, SA, AK, SB, BKc>(g, p, g.A, g.a_ps, g.B, g.b_ps, out, ldo, ss, bias, s);
            }
        } else {
            launch16<MT, SA, AK, SB, BKc>(g, p, g.A, g.a_ps, g.B, g.b_ps, out, ldo, ss, bias, s);
        }
    } else {
        launch16<MT, SA, AK, SB, BKc>(g, p, g.A, g.a_ps, g.B, g.b_ps, out, ldo, ss, bias, s);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (p.splits > 1) e = launch_splitk_reduce(g.M, g.N, p.splits, out, g.C, g.ldc, g.bias, s);
    return e;
}

// The combinations a dense layer needs (forward: both K-contiguous; weight
// gradient: both M/N-contiguous; input gradient: K- x N-contiguous).  `run`
// is false for a size query: returns whether the combination is supported.
hipError_t dispatch16(const GemmArgs &g, const Kind &kd, void *ws, size_t ws_bytes, hipStream_t s,
                      bool run, bool *supported) {
    *supported = true;
#define SNN_CASE(MT_, SA_, AK_, SB_, BK_)                                                            \
    if (kd.mt == MT_ && kd.sa == SA_ && g.a_kc == AK_ && kd.sb == SB_ && g.b_kc == BK_)              \
        return run ? run16<MT_, SA_, AK_, SB_, BK_>(g, kd, ws, ws_bytes, s) : hipSuccess;
    // currents x W^T
    SNN_CASE(MT_BF16, SRC_SPIKE, true, SRC_F32, true)
    SNN_CASE(MT_F16, SRC_SPIKE, true, SRC_H16, true)
    // dW = dI^T x, both transposed to K-contiguous (dI as bf16 planes)
    SNN_CASE(MT_BF16, SRC_PLANES, true, SRC_SPIKE, true)
    SNN_CASE(MT_BF16, SRC_H16, true, SRC_SPIKE, true)
    SNN_CASE(MT_F16, SRC_H16, true, SRC_SPIKE, true)
    // dW = dI^T x from the M/N-contiguous layouts
    SNN_CASE(MT_BF16, SRC_F32, false, SRC_SPIKE, false)
    SNN_CASE(MT_BF16, SRC_H16, false, SRC_SPIKE, false)
    SNN_CASE(MT_F16, SRC_H16, false, SRC_SPIKE, false)
    // dx = dI W with W transposed to K-contiguous
    SNN_CASE(MT_BF16, SRC_H16, true, SRC_F16X2, true)
    SNN_CASE(MT_BF16, SRC_F32, true, SRC_F16X2, true)
    SNN_CASE(MT_F16, SRC_H16, true, SRC_H16, true)
    // dx = dI W from W's own layout
    SNN_CASE(MT_BF16, SRC_H16, true, SRC_F16X2, false)
    SNN_CASE(MT_BF16, SRC_F32, true, SRC_F16X2, false)
    SNN_CASE(MT_F16, SRC_H16, true, SRC_H16, false)
    SNN_CASE(MT_BF16, SRC_H16, true, SRC_H16, false)
#undef SNN_CASE
    *supported = false;
    return hipErrorInvalidValue;
}

}  // namespace

bool gemm16_applies(const GemmArgs &g) {
    if (g.M < 1 || g.N < 1) return false;
    const Kind kd = classify(g.a_dtype, g.b_dtype);
    if (!kd.ok) return false;
    // a side below 64 wastes most of a tile: worth it only for one-pass pairs
    // (measured: fp32 x spikes skinny products are faster on the fp32 kernels)
    if ((g.M < 64 || g.N < 64) && parts_of(kd.sa) * parts_of(kd.sb) > 1) return false;
    bool sup = false;
    (void)dispatch16(g, kd, nullptr, 0, nullptr, false, &sup);  // a query: nothing launched
    return sup;
}

// Device-independent upper bound of the workspace any plan may use.
size_t gemm16_workspace_bytes(const GemmArgs &g) {
    if (!gemm16_applies(g) || g.K <= 0) return 0;
    const Kind kd = classify(g.a_dtype, g.b_dtype);
    const int ksteps = (g.K + BK - 1) / BK;
    size_t best = 0;
    for (int sh = 0; sh < kShapes; ++sh) {
        if (!shape_allowed(sh, kd)) continue;
        Plan16 p{};
        p.shape = sh;
        p.BM = kShapeBM[sh];
        p.BN = kShapeBN[sh];
        p.tiles_m = (g.M + p.BM - 1) / p.BM;
        p.tiles_n = (g.N + p.BN - 1) / p.BN;
        finish_plan(p, g.M, g.N, g.K, kd, g.a_kc, g.b_kc, max_splits(p.tiles_m * p.tiles_n, ksteps, (int64_t)g.M * g.N));
        best = max(best, p.plane_bytes + p.part_bytes);
    }
    return best;
}

hipError_t launch_gemm16(const GemmArgs &g, void *ws, size_t ws_bytes, hipStream_t s) {
    const Kind kd = classify(g.a_dtype, g.b_dtype);
    bool sup = false;
    return dispatch16(g, kd, ws, ws_bytes, s, true, &sup);
}

hipError_t launch_split_planes(const float *src, int64_t ld, int rows, int K, int ldp,
                               uint16_t *dst, hipStream_t s) {
    const int64_t n = (int64_t)rows * ldp;
    if (n <= 0) return hipSuccess;
    split_planes_kernel<<<(unsigned)((n + kThreads - 1) / kThreads), kThreads, 0, s>>>(src, ld, K,
                                                                                  ldp, n, dst);
    return hipGetLastError();
}

int gemm16_passes(const GemmArgs &g) {
    if (!gemm16_applies(g)) return 0;
    const Kind kd = classify(g.a_dtype, g.b_dtype);
    return parts_of(kd.sa) * parts_of(kd.sb);
}

}  // namespace snn

// ---- transposes that turn M/N-contiguous operands K-contiguous -------------
namespace snn {
namespace {

// dst[c][r] = src[r][c] through a 64x64 LDS tile (+1 column of padding).  A
// thread moves runs of 4 elements: it loads 4 consecutive columns of a source
// row and stores 4 consecutive rows of a destination row (16 threads cover
// one 64-element row), so both sides are 4-wide vector accesses when aligned;
// the LDS accesses of a wave fall on 64 distinct banks either way.  With
// PLANES, an fp32 source is written as three bf16 planes (dst + p*plane) of
// its exact split.
// perm_T > 0: destination index k takes source row (k % perm_T) *
// (rows / perm_T) + k / perm_T (rows = T B ordered [T][B] read as k = b T + t).
__device__ inline int src_row(int k, int rows, int perm_T) {
    return perm_T > 0 ? (k % perm_T) * (rows / perm_T) + k / perm_T : k;
}

template <typename T, bool PLANES>
__global__ __launch_bounds__(256) void transpose_kernel(int rows, int cols, const T *__restrict__ src,
                                                        int64_t lds_, void *__restrict__ dst,
                                                        int64_t ldd, int64_t plane, int perm_T) {
    __shared__ T tile[64][65];
    typedef uint16_t O;  // element type of the destination when PLANES
    const int r0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
    const int q = threadIdx.x & 15, g = threadIdx.x >> 4;
    {
        const int c = c0 + 4 * q;
        const bool vec = c + 4 <= cols && (lds_ & 3) == 0 &&
                         (((uintptr_t)src) & (4 * sizeof(T) - 1)) == 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int rl = g + 16 * j, r = r0 + rl;
            T v[4] = {T(0), T(0), T(0), T(0)};
            if (r < rows) {
                const T *p = src + (int64_t)src_row(r, rows, perm_T) * lds_ + c;
                if (vec) {
                    if constexpr (sizeof(T) == 4) {
                        const uint4 u = *reinterpret_cast<const uint4 *>(p);
                        v[0] = __uint_as_float(u.x); v[1] = __uint_as_float(u.y);
                        v[2] = __uint_as_float(u.z); v[3] = __uint_as_float(u.w);
                    } else {
                        const uint2 u = *reinterpret_cast<const uint2 *>(p);
                        v[0] = (T)(u.x & 0xffffu); v[1] = (T)(u.x >> 16);
                        v[2] = (T)(u.y & 0xffffu); v[3] = (T)(u.y >> 16);
                    }
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (c + e < cols) v[e] = p[e];
                }
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) tile[rl][4 * q + e] = v[e];
        }
    }
    __syncthreads();
    const int r = r0 + 4 * q;
    constexpr int OB = PLANES ? 2 : (int)sizeof(T);  // bytes per stored element
    const bool vec = r + 4 <= rows && (ldd & 3) == 0 && (!PLANES || (plane & 3) == 0) &&
                     (((uintptr_t)dst) & (4 * OB - 1)) == 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int cl = g + 16 * j, c = c0 + cl;
        if (c >= cols) continue;
        T v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = tile[4 * q + e][cl];
        const int64_t o = (int64_t)c * ldd + r;
        if constexpr (PLANES) {
            O *d16 = reinterpret_cast<O *>(dst);
#pragma unroll
            for (int p = 0; p < 3; ++p) {
                uint32_t h[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    uint32_t w[1] = {__float_as_uint((float)v[e])};
                    h[e] = part_of<SRC_F32, MT_BF16, 1>(w, 0, p);
                }
                O *d = d16 + p * plane + o;
                if (vec) {
                    *reinterpret_cast<uint2 *>(d) = make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16));
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (r + e < rows) d[e] = (O)h[e];
                }
            }
        } else {
            T *d = reinterpret_cast<T *>(dst) + o;
            if (vec) {
                if constexpr (sizeof(T) == 4) {
                    *reinterpret_cast<uint4 *>(d) =
                        make_uint4(__float_as_uint(v[0]), __float_as_uint(v[1]),
                                   __float_as_uint(v[2]), __float_as_uint(v[3]));
                } else {
                    *reinterpret_cast<uint2 *>(d) =
                        make_uint2((uint32_t)v[0] | ((uint32_t)v[1] << 16),
                                   (uint32_t)v[2] | ((uint32_t)v[3] << 16));
                }
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (r + e < rows) d[e] = v[e];
            }
        }
    }
}

// Bytes: dst[c][r] = src[r][c] through a 128 x 128 LDS tile.  Loads are 16
// bytes of a source row (8 threads per row); a thread then takes 4 columns
// of 16 rows (16 LDS words), regroups their bytes in registers and stores 4
// destination runs of 16 bytes (8 threads cover a 128-byte destination row).
// The tile's 132-byte row stride keeps the column-wise word reads of a wave
// within two rows per bank.
constexpr int kT8 = 128;       // tile side (bytes)
constexpr int kT8Row = 132;    // LDS row stride (bytes)
__global__ __launch_bounds__(256) void transpose_u8_kernel(int rows, int cols,
                                                           const uint8_t *__restrict__ src,
                                                           int64_t lds_, uint8_t *__restrict__ dst,
                                                           int64_t ldd, int perm_T) {
    __shared__ __attribute__((aligned(16))) uint32_t tile[kT8 * kT8Row / 4];
    const int r0 = blockIdx.y * kT8, c0 = blockIdx.x * kT8;
    const int t = threadIdx.x;
    {
        const int cc = (t & 7) * 16;
        const int gc = c0 + cc;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int r = (t >> 3) + 32 * i, gr = r0 + r;
            uint32_t w[4] = {0u, 0u, 0u, 0u};
            if (gr < rows) {
                const uint8_t *p = src + (int64_t)src_row(gr, rows, perm_T) * lds_ + gc;
                if (gc + 16 <= cols && (((uintptr_t)p) & 15) == 0) {
                    const uint4 v = *reinterpret_cast<const uint4 *>(p);
                    w[0] = v.x; w[1] = v.y; w[2] = v.z; w[3] = v.w;
                } else {
                    for (int e = 0; e < 16; ++e)
                        if (gc + e < cols) w[e / 4] |= (uint32_t)p[e] << (8 * (e % 4));
                }
            }
#pragma unroll
            for (int q = 0; q < 4; ++q) tile[(r * kT8Row + cc) / 4 + q] = w[q];
        }
    }
    __syncthreads();
    // thread: destination rows c0 + 4 cw .. + 3, source rows r0 + 16 rg .. + 15
    const int rg = t & 7, cw = t >> 3;
    uint32_t w[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) w[e] = tile[((16 * rg + e) * kT8Row) / 4 + cw];
    const int gr = r0 + 16 * rg;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int gc = c0 + 4 * cw + j;
        if (gc >= cols) continue;
        uint32_t o[4];
#pragma unroll
        for (int q = 0; q < 4; ++q)
            o[q] = ((w[4 * q] >> (8 * j)) & 0xffu) | (((w[4 * q + 1] >> (8 * j)) & 0xffu) << 8) |
                   (((w[4 * q + 2] >> (8 * j)) & 0xffu) << 16) |
                   (((w[4 * q + 3] >> (8 * j)) & 0xffu) << 24);
        uint8_t *q8 = dst + (int64_t)gc * ldd + gr;
        if (gr + 16 <= rows && (((uintptr_t)q8) & 15) == 0) {
            *reinterpret_cast<uint4 *>(q8) = make_uint4(o[0], o[1], o[2], o[3]);
        } else {
            for (int e = 0; e < 16; ++e)
                if (gr + e < rows) q8[e] = (uint8_t)(o[e / 4] >> (8 * (e % 4)));
        }
    }
}

}  // namespace

hipError_t launch_transpose(int rows, int cols, const void *src, int64_t ld_src, int elem_bytes,
                            void *dst, int64_t ld_dst, bool to_planes, int64_t plane,
                            hipStream_t s, int perm_T) {
    if (rows <= 0 || cols <= 0) return hipSuccess;
    if (perm_T < 0 || (perm_T > 0 && rows % perm_T != 0)) return hipErrorInvalidValue;
    dim3 grid((unsigned)((cols + 63) / 64), (unsigned)((rows + 63) / 64));
    if (to_planes) {
        if (elem_bytes != 4) return hipErrorInvalidValue;
        transpose_kernel<float, true><<<grid, 256, 0, s>>>(
            rows, cols, reinterpret_cast<const float *>(src), ld_src, dst, ld_dst, plane, perm_T);
    } else if (elem_bytes == 4) {
        transpose_kernel<float, false><<<grid, 256, 0, s>>>(
            rows, cols, reinterpret_cast<const float *>(src), ld_src, dst, ld_dst, 0, perm_T);
    } else if (elem_bytes == 2) {
        transpose_kernel<uint16_t, false><<<grid, 256, 0, s>>>(
            rows, cols, reinterpret_cast<const uint16_t *>(src), ld_src, dst, ld_dst, 0, perm_T);
    } else {
        const dim3 g8((unsigned)((cols + kT8 - 1) / kT8), (unsigned)((rows + kT8 - 1) / kT8));
        transpose_u8_kernel<<<g8, 256, 0, s>>>(rows, cols, reinterpret_cast<const uint8_t *>(src),
                                                 ld_src, reinterpret_cast<uint8_t *>(dst), ld_dst,
                                                 perm_T);
    }
    return hipGetLastError();
}

}  // namespace snn
