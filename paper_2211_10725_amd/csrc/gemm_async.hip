// Large single-part contractions on the 16-bit matrix cores with an
// asynchronous LDS pipeline:
//
//   C[M,N] = sum_k A[m][k] B[n][k] (+ bias[n]),  fp32 accumulate,
//
// A and B 16-bit values of the MFMA type (fp16, or bf16), both K-contiguous
// or both M/N-contiguous.  Spike operands (bytes, exact in either type) are
// first widened into the workspace.  Used for the big products of the
// half-precision network, where every product is one MFMA pass, and for the
// big products of spikes (or bf16 values) with an fp32 operand: that operand is held as three
// exact bf16 planes (hi, mid, lo; split into the workspace if given as fp32),
// and an item's k loop runs over the planes one after the other, the smallest
// first, each against the same spike tiles, accumulating in fp32 (three
// passes, every product exact).
//
// Tile 256 x 256 per workgroup of 8 wave64s (2 along M x 4 along N), 128 x 64
// per wave with v_mfma_f32_32x32x16_{f16,bf16}: two waves per SIMD, so one
// wave's MFMAs run while the other waits for its LDS reads (with one wave per
// SIMD the in-order issue leaves the matrix core idle during every read).  A
// wave reads 6 fragments per 8 MFMAs.  k-tiles of 64 are copied straight from
// global memory into two LDS stages (global_load_lds_dwordx4: lane i of a wave
// writes the 16 bytes at M0 + 16 i); the next tile is in flight while the
// current one is multiplied, and without registers.  Every row of a copy is
// 128 contiguous bytes.  Each stage of an operand is [256 rows][8 chunks of 8
// values] with chunk c of row r stored at slot c ^ swz(r),
// swz(r) = ((r >> 1) & 7) ^ ((r & 1) << 2): 8 consecutive rows of one chunk
// fall in 8 distinct 16-byte bank groups of a 128-byte line, and 16
// consecutive rows in 16 distinct groups of a 256-byte line (free of bank
// conflicts whether an LDS read serves 8 or 16 lanes at a time).  Every stage
// is its own LDS object, and the wait for a stage plus the workgroup barrier
// are one asm statement with a memory clobber: the compiler keeps the LDS
// reads after it.
//
// K must be a multiple of 8 (a 16-byte chunk is all in range or all out); the
// chunks past K of the last k-tile are loaded from column 0 and zeroed before
// the multiply.  Rows past M (N) load row M-1 (N-1) and are not stored.
#include <type_traits>

#include "snn_internal.hpp"

namespace snn {
namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) void lds_void;
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 512;  // 8 waves
constexpr int kTile = 256;                 // BM = BN
constexpr int kKT = 64;                    // k-tile
constexpr int kStage = kTile * kKT;        // 16-bit values per operand and stage (32 KiB)
constexpr int kGroupM = 4;                 // tile rows per group of the tile order

constexpr int MT_BF16 = 0;

__device__ inline int swz(int r) { return ((r >> 1) & 7) ^ ((r & 1) << 2); }
constexpr int MT_F16 = 1;

// one LDS object per stage: A tile, then B tile
__shared__ __attribute__((aligned(1024))) uint16_t g_s0[2 * kStage], g_s1[2 * kStage];

// The bias vector, staged once per workgroup: the epilogue reads its values
// from LDS, so no global load is pending when the next item starts (a global
// load there made the compiler wait for every store of the previous tile
// before the next item's first copies).  Layers with bias take this kernel
// only up to kBiasLds outputs.
constexpr int kBiasLds = 8192;
__shared__ float g_bias[kBiasLds];

template <int S>
__device__ inline uint16_t *stage_a() {
    if constexpr (S == 0) return g_s0;
    else return g_s1;
}
template <int S>
__device__ inline uint16_t *stage_b() { return stage_a<S>() + kStage; }

template <int MT>
__device__ inline floatx16 mfma32(const u32x4 &a, const u32x4 &b, const floatx16 &c) {
    if constexpr (MT == MT_F16)
        return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(half8, a),
                                                      __builtin_bit_cast(half8, b), c, 0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                       __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// Copies of one operand tile into a stage.  Wave w, copy j (of 4) fills
// stage bytes [(4 w + j) KiB, +1 KiB): row 8 (4 w + j) + lane / 8 of the tile,
// slot lane % 8, i.e. chunk c = (lane % 8) ^ swz(row); 8 consecutive lanes
// read one row's 128 contiguous bytes.  The per-thread row pointers (row
// clamped to the operand) and chunk offsets are fixed for the whole k loop; a
// chunk past K reads column 0 instead (zeroed before use).
struct TileCopyKC {
    const uint16_t *row[4];
    int c8[4];  // 8 * chunk

    __device__ inline void init(const uint16_t *X, int64_t ld, int rows, int r0) {
        const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int r = (4 * w + j) * 8 + (lane >> 3);
            c8[j] = 8 * ((lane & 7) ^ swz(r));
            row[j] = X + (int64_t)min(r0 + r, rows - 1) * ld;
        }
    }
    // off: element offset of the plane to copy from (0 for a one-part operand)
    __device__ inline void copy(int k0, int K, uint16_t *stage, int64_t off) const {
        // wave-uniform, so the LDS destinations are scalar (M0 set from SGPRs)
        const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int k = k0 + c8[j];
            __builtin_amdgcn_global_load_lds(row[j] + off + (k < K ? k : 0),
                                             (lds_void *)(stage + (4 * w + j) * 512), 16, 0, 0);
        }
    }
};

// M/N-contiguous operand ([k][row] in memory: dL/dI and the spikes in the
// weight gradient dW = dI^T x, K = T*B).  A stage holds [64 k-rows][256 rows]
// (512 bytes per k-row); 16-byte chunk c (rows 8c .. 8c + 7) of k-row k is
// stored at slot c ^ mn_swz(k).  Wave w, copy j fills stage bytes
// [(4 w + j) KiB, +1 KiB): k-rows 8 w + 2 j + lane / 32, slot lane % 32; the
// 32 lanes of a k-row read its 512 contiguous bytes.  k-rows past the end read
// the last one (zeroed before use); chunks past the last row read the last
// chunk (not stored).  Needs rows % 8 == 0.
__device__ inline int mn_swz(int k) { return 2 * ((k & 3) | ((k & 1) << 2)); }

struct TileCopyMN {
    const uint16_t *X;
    int64_t ld;
    int col[2];  // first row of the chunk this thread copies, for j even / odd
    int kr0;     // k-row of copy 0 within the tile

    __device__ inline void init(const uint16_t *X_, int64_t ld_, int rows, int r0) {
        const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
        X = X_;
        ld = ld_;
        kr0 = 8 * w + (lane >> 5);
#pragma unroll
        for (int jj = 0; jj < 2; ++jj)
            col[jj] = min(r0 + 8 * ((lane & 31) ^ mn_swz(kr0 + 2 * jj)), rows - 8);
    }
    __device__ inline void copy(int k0, int K, uint16_t *stage, int64_t off) const {
        // wave-uniform, so the LDS destinations are scalar (M0 set from SGPRs)
        const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int k = min(k0 + kr0 + 2 * j, K - 1);
            __builtin_amdgcn_global_load_lds(X + off + (int64_t)k * ld + col[j & 1],
                                             (lds_void *)(stage + (4 * w + j) * 512), 16, 0, 0);
        }
    }
};

template <bool MN>
using TileCopy = typename std::conditional<MN, TileCopyMN, TileCopyKC>::type;

// Wait until this thread's copies of the stage to multiply have landed (the
// only ones in flight), then the workgroup barrier: every wave's copies of
// that stage are in LDS, and every wave has finished reading the other stage,
// which the next copies overwrite.
__device__ inline void stage_barrier() { asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory"); }
// The first step of an item after a whole tile was stored through LDS: the
// 32 row stores of that epilogue were issued after this item's first
// copies, and vector memory operations complete in issue order, so waiting
// until at most 32 are outstanding waits for the copies only and leaves the
// stores draining under the first multiply.
__device__ inline void stage_barrier_after_stores() {
    asm volatile("s_waitcnt vmcnt(32)\n\ts_barrier" ::: "memory");
}

// LDS byte address of a stage element
__device__ inline uint32_t lds_addr(const uint16_t *p) {
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) uint16_t *)p;
}

// The fragment reads are issued as asm: the compiler's own wait insertion
// cannot tell the stages apart and would wait for every copy in flight
// before any LDS read.  The asm waits in multiply_stage name the fragments
// as operands, so no MFMA that uses them is scheduled before the data has
// arrived (LDS returns in order).
__device__ inline void lds_read(u32x4 &v, uint32_t addr) {
    asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(addr));
}

// LDS address of fragment i of k16 step ks: A fragments i = 0..3 (rows
// wm * 128 + 32 i), B fragments i = 4, 5 (rows wn * 64 + 32 (i - 4)).
template <int S>
__device__ inline uint32_t frag_addr(int wm, int wn, int ks, int i) {
    const int lane = threadIdx.x & 63;
    const int c = 2 * ks + (lane >> 5);
    const uint16_t *stage = i < 4 ? stage_a<S>() : stage_b<S>();
    const int r = (i < 4 ? wm * 128 + i * 32 : wn * 64 + (i - 4) * 32) + (lane & 31);
    return lds_addr(stage + r * kKT + (c ^ swz(r)) * 8);
}

// The 32 MFMAs of the four k16 steps of a stage.  A wave covers rows
// wm * 128 + [0, 128) and columns wn * 64 + [0, 64).  The 6 fragment reads of
// step ks + 1 are issued one by one between the 8 MFMAs of step ks
// (scheduling barriers keep that order), so the wave issues them while the
// matrix core is busy instead of stalling on them between steps.
template <int MT, int S, typename Issue>
__device__ inline void multiply_stage(floatx16 (&acc)[4][2], int wm, int wn, int kvalid,
                                      const Issue &issue) {
    const int half = (threadIdx.x & 63) >> 5;
    u32x4 f[2][6];
#pragma unroll
    for (int i = 0; i < 6; ++i) lds_read(f[0][i], frag_addr<S>(wm, wn, 0, i));
    __builtin_amdgcn_sched_barrier(0);
    issue();
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
        u32x4(&cur)[6] = f[ks & 1];
        u32x4(&nxt)[6] = f[(ks + 1) & 1];
        asm volatile("s_waitcnt lgkmcnt(0)"
                     : "+v"(cur[0]), "+v"(cur[1]), "+v"(cur[2]), "+v"(cur[3]), "+v"(cur[4]),
                       "+v"(cur[5]));
        if (kvalid < kKT) {
            const uint32_t m = 8 * (2 * ks + half) < kvalid ? 0xffffffffu : 0u;
#pragma unroll
            for (int i = 0; i < 6; ++i) cur[i] &= m;
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const int i = q >> 1, j = q & 1;
            acc[i][j] = mfma32<MT>(cur[i], cur[4 + j], acc[i][j]);
            __builtin_amdgcn_sched_barrier(0);
            if (ks + 1 < 4 && q < 6) {
                lds_read(nxt[q], frag_addr<S>(wm, wn, ks + 1, q));
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    }
}

// M/N-contiguous stages: a fragment is two transposing reads.  Within each 16
// lanes, ds_read_b64_tr_b16 hands lane i element e of lane 4 e + i / 4's
// 4-element run (position i % 4).  Lane L of 16-lane group g points at k-row
// kb + L / 4 and rows j0 + 4 (L % 4), j0 = fragment row + 16 (g & 1), kb =
// 16 ks + 8 (g >> 1) + 4 r: lane i of the group receives k = kb .. kb + 3 of
// row j0 + i, and reads r = 0, 1 make the 8 k-contiguous values of the MFMA
// operand.  A read's 16-lane group covers 4 k-rows of 32 bytes each: with the
// chunk slots XORed by mn_swz(k) (k mod 4 -> 32-byte slot XOR 0, 5, 2, 7),
// the 4 k-rows of a group fall on distinct banks of a 128-byte line and the 8
// of two groups on distinct banks of a 256-byte line.  k mod 4 is fixed per
// lane, so step ks and read r are constant offsets from the lane's address.
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ inline void lds_read_tr(u32x2 &v, uint32_t addr) {
    asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(v) : "v"(addr));
}

template <int S>
__device__ inline uint32_t frag_addr_mn(int wm, int wn, int i) {
    const int lane = threadIdx.x & 63, g = lane >> 4, L = lane & 15;
    const uint16_t *stage = i < 4 ? stage_a<S>() : stage_b<S>();
    const int row = (i < 4 ? wm * 128 + i * 32 : wn * 64 + (i - 4) * 32) + 16 * (g & 1) + 4 * (L & 3);
    const int kr = 8 * (g >> 1) + (L >> 2);
    return lds_addr(stage + kr * kTile + ((row >> 3) ^ mn_swz(kr)) * 8 + (row & 7));
}

template <int MT, int S, typename Issue>
__device__ inline void multiply_stage_mn(floatx16 (&acc)[4][2], int wm, int wn, int kvalid,
                                         const Issue &issue) {
    const int half = (threadIdx.x & 63) >> 5;
    uint32_t base[6];
#pragma unroll
    for (int i = 0; i < 6; ++i) base[i] = frag_addr_mn<S>(wm, wn, i);
    u32x2 f[2][6][2];
#pragma unroll
    for (int i = 0; i < 6; ++i)
#pragma unroll
        for (int r = 0; r < 2; ++r) lds_read_tr(f[0][i][r], base[i] + r * 4 * kTile * 2);
    __builtin_amdgcn_sched_barrier(0);
    issue();
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
        u32x2(&cur)[6][2] = f[ks & 1];
        u32x2(&nxt)[6][2] = f[(ks + 1) & 1];
        asm volatile("s_waitcnt lgkmcnt(0)"
                     : "+v"(cur[0][0]), "+v"(cur[0][1]), "+v"(cur[1][0]), "+v"(cur[1][1]),
                       "+v"(cur[2][0]), "+v"(cur[2][1]), "+v"(cur[3][0]), "+v"(cur[3][1]),
                       "+v"(cur[4][0]), "+v"(cur[4][1]), "+v"(cur[5][0]), "+v"(cur[5][1]));
        if (kvalid < kKT) {
            const uint32_t m = 8 * (2 * ks + half) < kvalid ? 0xffffffffu : 0u;
#pragma unroll
            for (int i = 0; i < 6; ++i) {
                cur[i][0] &= m;
                cur[i][1] &= m;
            }
        }
        u32x4 op[6];
#pragma unroll
        for (int i = 0; i < 6; ++i) op[i] = __builtin_shufflevector(cur[i][0], cur[i][1], 0, 1, 2, 3);
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const int i = q >> 1, j = q & 1;
            acc[i][j] = mfma32<MT>(op[i], op[4 + j], acc[i][j]);
            __builtin_amdgcn_sched_barrier(0);
            if (ks + 1 < 4 && q < 6) {
#pragma unroll
                for (int r = 0; r < 2; ++r)
                    lds_read_tr(nxt[q][r], base[q] + ((ks + 1) * 16 + r * 4) * kTile * 2);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    }
}

// The stage's first fragment reads go out before issue() (the copies of the
// next k-tile into the other stage), so their latency covers the copies'
// address arithmetic and issue.
template <int MT, bool MN, int S, typename Issue>
__device__ inline void multiply(floatx16 (&acc)[4][2], int wm, int wn, int kvalid,
                                const Issue &issue) {
    if constexpr (MN) multiply_stage_mn<MT, S>(acc, wm, wn, kvalid, issue);
    else multiply_stage<MT, S>(acc, wm, wn, kvalid, issue);
}

// ---- storing a 256 x 256 fp32 result tile ------------------------------------
// In the 32x32 MFMA block (i, q) of wave (wm, wn), a lane holds column
// wn * 64 + 32 q + (lane & 31) and, in register r, row wm * 128 + 32 i +
// 8 (r / 4) + 4 (lane / 32) + r % 4 of the tile.  A scaled operand's power of
// two is divided out exactly (multiplication by its exact reciprocal).

// Directly from the registers: every store instruction writes two 128-byte
// row pieces (for C rows that are not 16-byte aligned).
__device__ inline void store_tile_direct(const floatx16 (&acc)[4][2], float *Cz, int64_t ldc,
                                         int M, int N, int m0, int n0, int wm, int wn, float inv,
                                         const float (&bn)[2]) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            const int n = n0 + wn * 64 + q * 32 + (lane & 31);
            if (n >= N) continue;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int m = m0 + wm * 128 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
                if (m < M) Cz[(int64_t)m * ldc + n] = acc[i][q][r] * inv + bn[q];
            }
        }
}

// Through LDS (the second stage, free once every wave is past its last
// multiply): four passes of 64 tile rows.  In a pass the four waves that hold
// those rows write them into a [64][256] fp32 tile (column c of row R at
// c ^ 32 (R & 4 ? 1 : 0), so the two half-waves of a write fall on distinct
// banks), then every thread stores 16 contiguous bytes of a row: each store
// instruction writes one whole 1 KiB row of C.  Measured on the
// 51200 x 4096 products: a quarter of the store instructions of the direct
// epilogue and about a fifth of the kernel time at K = 784.
__device__ inline void store_tile_lds(const floatx16 (&acc)[4][2], float *Cz, int64_t ldc, int M,
                                      int N, int m0, int n0, int wm, int wn, float inv,
                                      const float (&bn)[2]) {
    float *t = reinterpret_cast<float *>(stage_a<1>());  // 64 KiB: [64][256]
    const int lane = threadIdx.x & 63;
    const bool full = m0 + kTile <= M && n0 + kTile <= N;
#pragma unroll
    for (int pass = 0; pass < 4; ++pass) {
        __syncthreads();  // the stage (or the previous pass) is no longer read
        if (wm == pass / 2) {
#pragma unroll
            for (int ii = 0; ii < 2; ++ii) {
                const int i = 2 * (pass & 1) + ii;
#pragma unroll
                for (int q = 0; q < 2; ++q) {
                    const int c = wn * 64 + q * 32 + (lane & 31);
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const int R = ii * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
                        t[R * 256 + (c ^ ((R & 4) << 3))] = acc[i][q][r] * inv + bn[q];
                    }
                }
            }
        }
        __syncthreads();
        const int c = 4 * lane, n = n0 + c;
        float4 v[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            const int R = (threadIdx.x >> 6) + 8 * k;  // one row per wave and k
            v[k] = *reinterpret_cast<const float4 *>(&t[R * 256 + (c ^ ((R & 4) << 3))]);
        }
        float *row = Cz + (int64_t)(m0 + 64 * pass + (threadIdx.x >> 6)) * ldc + n;
        if (full) {
#pragma unroll
            for (int k = 0; k < 8; ++k) *reinterpret_cast<float4 *>(row + 8 * k * ldc) = v[k];
        } else {
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                if (m0 + 64 * pass + (threadIdx.x >> 6) + 8 * k >= M) continue;
                float *dst = row + 8 * k * ldc;
                if (n + 3 < N) {
                    *reinterpret_cast<float4 *>(dst) = v[k];
                } else {
                    if (n < N) dst[0] = v[k].x;
                    if (n + 1 < N) dst[1] = v[k].y;
                    if (n + 2 < N) dst[2] = v[k].z;
                }
            }
        }
    }
}

// Work item i of the launch (a tile and a K split) for persistent workgroup
// w of G: the items are cut into kXcds contiguous ranges, one per XCD
// (workgroup w runs on XCD w % kXcds), and the XCD's workgroups take the
// items of its range in turn, so the tiles in flight on one XCD are
// neighbours (they share operand panels in that XCD's L2).
__device__ inline int persistent_item(int w, int G, int total, int j) {
    const int xcd = w % kXcds, lw = w / kXcds;
    const int gx = G / kXcds + (xcd < G % kXcds ? 1 : 0);  // workgroups on this XCD
    const int per = total / kXcds, rem = total % kXcds;
    const int beg = xcd < rem ? xcd * (per + 1) : rem * (per + 1) + (xcd - rem) * per;
    const int cnt = per + (xcd < rem ? 1 : 0);
    const int k = lw + j * gx;
    return k < cnt ? beg + k : -1;
}

// Persistent: gridDim.x workgroups (one per CU) loop over the work items.
// The first k-tile of a workgroup's next item is copied into stage 0 before
// the current item's results are stored (through stage 1) (stage 0 was last read before the
// barrier of the current item's final k-tile), so that latency overlaps the
// stores.  P = 3: one operand is three bf16 planes (a_ps / b_ps elements
// apart, the other's stride 0); step v = p nk + kk of an item multiplies
// k-tile kk of plane 2 - p (lo, then mid, then hi).
template <int MT, bool MN, int P>
__global__ __launch_bounds__(kThreads, 1) void gemm_async_kernel(
    int M, int N, int K, int k_chunk, int tiles_n, int tiles, int total,
    const uint16_t *__restrict__ A, int64_t lda, const uint16_t *__restrict__ B, int64_t ldb,
    float *__restrict__ C, int64_t ldc, int64_t split_stride, const float *__restrict__ bias,
    const float *__restrict__ c_div, int64_t a_ps, int64_t b_ps) {
    const int wave = threadIdx.x >> 6, wm = wave & 1, wn = wave >> 1;
    const int lane = threadIdx.x & 63;
    const float inv = c_div ? 1.f / c_div[0] : 1.f;
    // rows of C (and of every split's partial sums) start on 16 bytes
    const bool wide_stores = ((uintptr_t)C & 15) == 0 && (ldc & 3) == 0 && (split_stride & 3) == 0;
    int item = persistent_item(blockIdx.x, gridDim.x, total, 0);
    if (item < 0) return;
    if (bias) {
        for (int i = threadIdx.x; i < N; i += kThreads) g_bias[i] = bias[i];
        __syncthreads();
    }
    TileCopy<MN> ca, cb;
    auto setup = [&](int it, int &m0, int &n0, int &zk, int &kbeg, int &kend, int &nk) {
        zk = it / tiles;
        // Tiles in groups of kGroupM tile rows, column by column within a
        // group: the 32 tiles an XCD's workgroups hold at once then span 4
        // rows and 8 columns, 12 operand panels instead of the 18 of 2 full
        // rows of 16 (measured: 8 % less time on the 51200 x 4096 x 4096
        // products than row-major tiles, 4 % less than groups of 8).
        const int tile = it % tiles;
        const int grp = tile / (kGroupM * tiles_n), first = grp * kGroupM;
        const int gm = min(kGroupM, tiles / tiles_n - first), local = tile % (kGroupM * tiles_n);
        m0 = (first + local % gm) * kTile;
        n0 = (local / gm) * kTile;
        kbeg = zk * k_chunk;
        kend = min(K, kbeg + k_chunk);
        nk = (kend - kbeg + kKT - 1) / kKT;  // >= 1
        ca.init(A, lda, M, m0);
        cb.init(B, ldb, N, n0);
    };
    // plane offsets of the first step (part 0: the last plane)
    const int64_t a_off0 = (P - 1) * a_ps, b_off0 = (P - 1) * b_ps;
    int m0, n0, zk, kbeg, kend, nk;
    bool stores_pending = false;  // the previous item stored a whole tile through LDS
    setup(item, m0, n0, zk, kbeg, kend, nk);
    ca.copy(kbeg, kend, stage_a<0>(), a_off0);
    cb.copy(kbeg, kend, stage_b<0>(), b_off0);
    for (int j = 0; item >= 0; ++j) {
        floatx16 acc[4][2];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int q = 0; q < 2; ++q)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[i][q][r] = 0.f;
        // Step tt of this item: part cp, k-tile ck (P = 1: k-tile tt).  The
        // loop runs an even number of steps; with an odd number of steps the
        // last one only waits at the barrier.
        const int nv = P * nk, nv2 = (nv + 1) & ~1;
        int cp = 0, ck = 0;
        for (int t = 0; t < nv2; t += 2) {
#define SNN_ASYNC_STEP(S, NEXT)                                                             \
    {                                                                                       \
        const int tt = t + (S);                                                             \
        if (tt == 0 && stores_pending)                                                      \
            stage_barrier_after_stores();                                                   \
        else                                                                                \
            stage_barrier();                                                                \
        if (tt < nv) {                                                                      \
            int np = 0, nkk = tt + 1, kc = tt;                                              \
            if constexpr (P > 1) {                                                          \
                kc = ck;                                                                    \
                np = cp;                                                                    \
                nkk = ck + 1;                                                               \
                if (nkk == nk) {                                                            \
                    nkk = 0;                                                                \
                    ++np;                                                                   \
                }                                                                           \
            }                                                                               \
            multiply<MT, MN, S>(acc, wm, wn, kend - (kbeg + kKT * kc), [&] {                \
                if (tt + 1 < nv) {                                                          \
                    ca.copy(kbeg + kKT * nkk, kend, stage_a<NEXT>(), (P - 1 - np) * a_ps);  \
                    cb.copy(kbeg + kKT * nkk, kend, stage_b<NEXT>(), (P - 1 - np) * b_ps);  \
                }                                                                           \
            });                                                                             \
            if constexpr (P > 1) {                                                          \
                cp = np;                                                                    \
                ck = nkk;                                                                   \
            }                                                                               \
        }                                                                                   \
    }
            SNN_ASYNC_STEP(0, 1)
            SNN_ASYNC_STEP(1, 0)
#undef SNN_ASYNC_STEP
        }
        const int m0c = m0, n0c = n0, zkc = zk;
        float bn[2];
#pragma unroll
        for (int q = 0; q < 2; ++q)
            bn[q] = bias ? g_bias[min(n0c + wn * 64 + q * 32 + (lane & 31), N - 1)] : 0.f;
        // the next item's first k-tile, in flight during the stores below
        item = persistent_item(blockIdx.x, gridDim.x, total, j + 1);
        if (item >= 0) setup(item, m0, n0, zk, kbeg, kend, nk);
        ca.copy(kbeg, kend, stage_a<0>(), a_off0);
        cb.copy(kbeg, kend, stage_b<0>(), b_off0);
        float *Cz = C + (int64_t)zkc * split_stride;
        if (wide_stores)
            store_tile_lds(acc, Cz, ldc, M, N, m0c, n0c, wm, wn, inv, bn);
        else
            store_tile_direct(acc, Cz, ldc, M, N, m0c, n0c, wm, wn, inv, bn);
        stores_pending = wide_stores && m0c + kTile <= M && n0c + kTile <= N;
    }
    // the workgroup's LDS must not be released with copies into it in flight
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

// Spike bytes widened to the 16-bit MFMA type: dst[r][k] (ld K) from
// src[r * lds + k]; byte values are exact in fp16 and bf16.
template <int MT>
__global__ __launch_bounds__(kThreads) void widen_kernel(int64_t rows, int K, const uint8_t *__restrict__ src,
                                                         int64_t lds, uint16_t *__restrict__ dst) {
    const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;  // one 8-value chunk
    const int cpr = K / 8;
    if (i >= rows * cpr) return;
    const int64_t r = i / cpr;
    const int k0 = (int)(i - r * cpr) * 8;
    uint32_t h[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const float v = (float)src[r * lds + k0 + e];
        if constexpr (MT == MT_F16) h[e] = __builtin_bit_cast(uint16_t, (_Float16)v);
        else h[e] = __float_as_uint(v) >> 16;
    }
    *reinterpret_cast<uint4 *>(dst + r * K + k0) =
        make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16));
}

unsigned blocks(int64_t n) { return (unsigned)((n + kThreads - 1) / kThreads); }

// bf16 planes of an operand: an fp32 array (split into the workspace) or
// one already split into three planes
bool planar(int t) { return t == SNN_F32 || t == kPlanes3; }

// MFMA type of an operand pair, or -1: fp16 for spikes/fp16, bf16 for
// spikes/bf16 and for spikes or bf16 values against three bf16 planes (a
// product of two bf16 values is exact in fp32).
int mfma_type(int a, int b) {
    auto f16ish = [](int t) { return t == SNN_U8 || t == SNN_F16; };
    auto bf16ish = [](int t) { return t == SNN_U8 || t == SNN_BF16; };
    if ((planar(a) && bf16ish(b)) || (bf16ish(a) && planar(b))) return MT_BF16;
    if (a == SNN_U8 && b == SNN_U8) return MT_F16;
    if (f16ish(a) && f16ish(b)) return MT_F16;
    if (bf16ish(a) && bf16ish(b)) return MT_BF16;
    return -1;
}

struct AsyncPlan {
    int tiles_m, tiles_n, splits, k_chunk, parts;
    size_t a_bytes, b_bytes;  // widened spike operands, or the planes of an fp32 operand
    size_t part_bytes;        // split-K partial sums
};

// 16-bit elements per plane row of an fp32 operand split in its own layout
// ([rows][K] K-contiguous, [K][rows] M/N-contiguous): rows start on 16 bytes
int64_t plane_ld(const GemmArgs &g, int rows) { return g.a_kc ? (g.K + 7) / 8 * 8 : (rows + 7) / 8 * 8; }
int64_t plane_rows(const GemmArgs &g, int rows) { return g.a_kc ? rows : g.K; }

AsyncPlan plan_async(const GemmArgs &g) {
    AsyncPlan p{};
    p.tiles_m = (g.M + kTile - 1) / kTile;
    p.tiles_n = (g.N + kTile - 1) / kTile;
    p.parts = planar(g.a_dtype) || planar(g.b_dtype) ? 3 : 1;
    const int tiles = p.tiles_m * p.tiles_n;
    const int nk = (g.K + kKT - 1) / kKT;
    int S = 1;
    const int cus = 256;  // one workgroup per CU; MI355X has 256 CUs
    if (tiles < cus) S = max(1, min(min(cus / tiles, p.parts * nk / 16), 64));
    const int per = (nk + S - 1) / S;
    p.k_chunk = per * kKT;
    p.splits = (g.K + p.k_chunk - 1) / p.k_chunk;
    auto operand = [&](int t, int rows) -> size_t {
        if (t == SNN_U8) return align_up((size_t)rows * g.K * 2);
        if (t == SNN_F32) return align_up((size_t)3 * plane_rows(g, rows) * plane_ld(g, rows) * 2);
        return 0;
    };
    p.a_bytes = operand(g.a_dtype, g.M);
    p.b_bytes = operand(g.b_dtype, g.N);
    p.part_bytes = p.splits > 1 ? align_up((size_t)p.splits * g.M * g.N * sizeof(float)) : 0;
    return p;
}

}  // namespace

bool gemm_async_applies(const GemmArgs &g) {
    // both operands K-contiguous, or both M/N-contiguous
    if (!g.allow_split || g.a_kc != g.b_kc) return false;
    if (mfma_type(g.a_dtype, g.b_dtype) < 0) return false;
    if (g.K % 8 != 0 || g.K < 256 || g.M < kTile || g.N < kTile) return false;
    if (g.bias && g.N > kBiasLds) return false;
    if (!g.a_kc && (g.M % 8 != 0 || g.N % 8 != 0)) return false;
    if (g.a_dtype != SNN_U8 && g.a_dtype != SNN_F32 && g.lda % 8 != 0) return false;
    if (g.b_dtype != SNN_U8 && g.b_dtype != SNN_F32 && g.ldb % 8 != 0) return false;
    if (g.a_dtype == kPlanes3 && g.a_ps % 8 != 0) return false;
    if (g.b_dtype == kPlanes3 && g.b_ps % 8 != 0) return false;
    if (planar(g.a_dtype) || planar(g.b_dtype)) {
        // three passes: the pooling epilogue of a convolution stays with the
        // kernels that have it; enough 256 x 256 tiles to fill the device
        if (g.pool_hw > 0 || g.c_div) return false;
        const AsyncPlan p = plan_async(g);
        if (p.tiles_m * p.tiles_n * p.splits < 192) return false;
        return (double)g.M * g.N * g.K >= 4294967296.0;
    }
    // large enough to fill the device with 256 x 256 tiles (K split as needed)
    return (double)g.M * g.N * g.K >= 1073741824.0;
}

size_t gemm_async_workspace_bytes(const GemmArgs &g) {
    if (!gemm_async_applies(g)) return 0;
    const AsyncPlan p = plan_async(g);
    return p.a_bytes + p.b_bytes + p.part_bytes;
}

hipError_t launch_gemm_async(const GemmArgs &g, void *ws, size_t ws_bytes, hipStream_t s) {
    const AsyncPlan p = plan_async(g);
    const int mt = mfma_type(g.a_dtype, g.b_dtype);
    if (p.a_bytes + p.b_bytes + p.part_bytes > 0 &&
        (ws == nullptr || ws_bytes < p.a_bytes + p.b_bytes + p.part_bytes))
        return hipErrorInvalidValue;
    char *w = reinterpret_cast<char *>(ws);
    const uint16_t *A = reinterpret_cast<const uint16_t *>(g.A);
    const uint16_t *B = reinterpret_cast<const uint16_t *>(g.B);
    int64_t lda = g.lda, ldb = g.ldb, a_ps = g.a_dtype == kPlanes3 ? g.a_ps : 0,
            b_ps = g.b_dtype == kPlanes3 ? g.b_ps : 0;
    const bool mn = !g.a_kc;
    // a spike operand widened in its own layout: [rows][K] or [K][rows]
    auto widen = [&](const void *src, int64_t ld, int rows, uint16_t *d) {
        const int r = mn ? g.K : rows, c = mn ? rows : g.K;
        const int64_t n = (int64_t)r * (c / 8);
        if (mt == MT_F16)
            widen_kernel<MT_F16><<<blocks(n), kThreads, 0, s>>>(r, c, reinterpret_cast<const uint8_t *>(src), ld, d);
        else
            widen_kernel<MT_BF16><<<blocks(n), kThreads, 0, s>>>(r, c, reinterpret_cast<const uint8_t *>(src), ld, d);
        return (int64_t)c;
    };
    // an fp32 operand split into three bf16 planes in its own layout
    auto split = [&](const void *src, int64_t ld, int rows, uint16_t *d, int64_t &ps) {
        const int64_t pr = plane_rows(g, rows), pl = plane_ld(g, rows);
        ps = pr * pl;
        return launch_split_planes(reinterpret_cast<const float *>(src), ld, (int)pr,
                                   mn ? rows : g.K, (int)pl, d, s) == hipSuccess ? pl : (int64_t)-1;
    };
    if (p.a_bytes) {
        uint16_t *d = reinterpret_cast<uint16_t *>(w);
        lda = g.a_dtype == SNN_F32 ? split(g.A, g.lda, g.M, d, a_ps) : widen(g.A, g.lda, g.M, d);
        A = d;
    }
    if (p.b_bytes) {
        uint16_t *d = reinterpret_cast<uint16_t *>(w + p.a_bytes);
        ldb = g.b_dtype == SNN_F32 ? split(g.B, g.ldb, g.N, d, b_ps) : widen(g.B, g.ldb, g.N, d);
        B = d;
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (lda < 0 || ldb < 0) return hipErrorInvalidValue;
    float *out = g.C;
    int64_t ldo = g.ldc, ss = 0;
    const float *bias = g.bias, *c_div = g.c_div;
    if (p.splits > 1) {
        out = reinterpret_cast<float *>(w + p.a_bytes + p.b_bytes);
        ldo = g.N;
        ss = (int64_t)g.M * g.N;
        bias = nullptr;
        c_div = nullptr;  // divided in the reduction
    }
    const int tiles = p.tiles_m * p.tiles_n, total = tiles * p.splits;
    // one persistent workgroup per compute unit (128 KiB of LDS each)
    const unsigned grid = (unsigned)min(total, device_cus());
    decltype(&gemm_async_kernel<MT_F16, false, 1>) kernel;
    if (p.parts == 3)
        kernel = mn ? gemm_async_kernel<MT_BF16, true, 3> : gemm_async_kernel<MT_BF16, false, 3>;
    else if (mt == MT_F16)
        kernel = mn ? gemm_async_kernel<MT_F16, true, 1> : gemm_async_kernel<MT_F16, false, 1>;
    else
        kernel = mn ? gemm_async_kernel<MT_BF16, true, 1> : gemm_async_kernel<MT_BF16, false, 1>;
    kernel<<<grid, kThreads, 0, s>>>(g.M, g.N, g.K, p.k_chunk, p.tiles_n, tiles, total, A, lda, B,
                                     ldb, out, ldo, ss, bias, c_div, a_ps, b_ps);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (p.splits > 1)
        e = launch_splitk_reduce(g.M, g.N, p.splits, out, g.C, g.ldc, g.bias, s, g.c_div);
    return e;
}

}  // namespace snn
