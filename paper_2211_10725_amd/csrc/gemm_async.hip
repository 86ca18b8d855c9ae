// Large single-part contractions on the 16-bit matrix cores with an
// asynchronous LDS pipeline:
//
//   C[M,N] = sum_k A[m][k] B[n][k] (+ bias[n]),  fp32 accumulate,
//
// A and B 16-bit values of the MFMA type (fp16, or bf16), both K-contiguous.
// Spike operands (bytes, exact in either type) are first widened into the
// workspace.  Used for the big products of the half-precision network, where
// every product is one MFMA pass.
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

constexpr int MT_BF16 = 0;

__device__ inline int swz(int r) { return ((r >> 1) & 7) ^ ((r & 1) << 2); }
constexpr int MT_F16 = 1;

// one LDS object per stage: A tile, then B tile
__shared__ __attribute__((aligned(1024))) uint16_t g_s0[2 * kStage], g_s1[2 * kStage];

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
struct TileCopy {
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
    __device__ inline void copy(int k0, int K, uint16_t *stage) const {
        const int w = threadIdx.x >> 6;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int k = k0 + c8[j];
            __builtin_amdgcn_global_load_lds(row[j] + (k < K ? k : 0),
                                             (lds_void *)(stage + (4 * w + j) * 512), 16, 0, 0);
        }
    }
};

// Wait until this thread's copies of the stage to multiply have landed (the
// only ones in flight), then the workgroup barrier: every wave's copies of
// that stage are in LDS, and every wave has finished reading the other stage,
// which the next copies overwrite.
__device__ inline void stage_barrier() { asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory"); }

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
template <int MT, int S>
__device__ inline void multiply_stage(floatx16 (&acc)[4][2], int wm, int wn, int kvalid) {
    const int half = (threadIdx.x & 63) >> 5;
    u32x4 f[2][6];
#pragma unroll
    for (int i = 0; i < 6; ++i) lds_read(f[0][i], frag_addr<S>(wm, wn, 0, i));
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
// the current item's results are stored (stage 0 was last read before the
// barrier of the current item's final k-tile), so that latency overlaps the
// stores.
template <int MT>
__global__ __launch_bounds__(kThreads, 1) void gemm_async_kernel(
    int M, int N, int K, int k_chunk, int tiles_n, int tiles, int total,
    const uint16_t *__restrict__ A, int64_t lda, const uint16_t *__restrict__ B, int64_t ldb,
    float *__restrict__ C, int64_t ldc, int64_t split_stride, const float *__restrict__ bias,
    const float *__restrict__ c_div) {
    const int wave = threadIdx.x >> 6, wm = wave & 1, wn = wave >> 1;
    const int lane = threadIdx.x & 63;
    const float inv = c_div ? 1.f / c_div[0] : 1.f;
    int item = persistent_item(blockIdx.x, gridDim.x, total, 0);
    if (item < 0) return;
    TileCopy ca, cb;
    auto setup = [&](int it, int &m0, int &n0, int &zk, int &kbeg, int &kend, int &nk) {
        zk = it / tiles;
        const int tile = it % tiles;
        m0 = (tile / tiles_n) * kTile;
        n0 = (tile % tiles_n) * kTile;
        kbeg = zk * k_chunk;
        kend = min(K, kbeg + k_chunk);
        nk = (kend - kbeg + kKT - 1) / kKT;  // >= 1
        ca.init(A, lda, M, m0);
        cb.init(B, ldb, N, n0);
    };
    int m0, n0, zk, kbeg, kend, nk;
    setup(item, m0, n0, zk, kbeg, kend, nk);
    ca.copy(kbeg, kend, stage_a<0>());
    cb.copy(kbeg, kend, stage_b<0>());
    for (int j = 0; item >= 0; ++j) {
        floatx16 acc[4][2];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int q = 0; q < 2; ++q)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[i][q][r] = 0.f;
        // k-tile t of this item.  The loop runs an even number of tiles; a
        // tile past the end re-copies the last one and is multiplied fully
        // masked.
        const int nk2 = (nk + 1) & ~1;
#define SNN_KTILE(t) (kbeg + kKT * min((t), nk - 1))
        for (int t = 0; t < nk2; t += 2) {
#define SNN_ASYNC_STEP(S, NEXT)                                                             \
    {                                                                                       \
        const int tt = t + (S);                                                             \
        stage_barrier();                                                                    \
        if (tt + 1 < nk2) {                                                                 \
            ca.copy(SNN_KTILE(tt + 1), kend, stage_a<NEXT>());                              \
            cb.copy(SNN_KTILE(tt + 1), kend, stage_b<NEXT>());                              \
        }                                                                                   \
        multiply_stage<MT, S>(acc, wm, wn, kend - (kbeg + kKT * tt));                       \
    }
            SNN_ASYNC_STEP(0, 1)
            SNN_ASYNC_STEP(1, 0)
#undef SNN_ASYNC_STEP
        }
#undef SNN_KTILE
        // the next item's first k-tile, in flight during the stores below
        const int m0c = m0, n0c = n0, zkc = zk;
        item = persistent_item(blockIdx.x, gridDim.x, total, j + 1);
        if (item >= 0) {
            setup(item, m0, n0, zk, kbeg, kend, nk);
            ca.copy(kbeg, kend, stage_a<0>());
            cb.copy(kbeg, kend, stage_b<0>());
        }
        // 32x32 block: lane holds column (lane & 31); register r holds row
        // 8*(r/4) + 4*(lane/32) + r%4.  A scaled operand's power of two is
        // divided out exactly (multiplication by its exact reciprocal).
        float *Cz = C + (int64_t)zkc * split_stride;
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int q = 0; q < 2; ++q) {
                const int n = n0c + wn * 64 + q * 32 + (lane & 31);
                if (n >= N) continue;
                const float bn = bias ? bias[n] : 0.f;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int m = m0c + wm * 128 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
                    if (m < M) Cz[(int64_t)m * ldc + n] = acc[i][q][r] * inv + bn;
                }
            }
    }
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

// MFMA type of an operand pair, or -1: fp16 for spikes/fp16, bf16 for spikes/bf16.
int mfma_type(int a, int b) {
    auto f16ish = [](int t) { return t == SNN_U8 || t == SNN_F16; };
    auto bf16ish = [](int t) { return t == SNN_U8 || t == SNN_BF16; };
    if (a == SNN_U8 && b == SNN_U8) return MT_F16;
    if (f16ish(a) && f16ish(b)) return MT_F16;
    if (bf16ish(a) && bf16ish(b)) return MT_BF16;
    return -1;
}

struct AsyncPlan {
    int tiles_m, tiles_n, splits, k_chunk;
    size_t a_bytes, b_bytes;  // widened spike operands
    size_t part_bytes;        // split-K partial sums
};

AsyncPlan plan_async(const GemmArgs &g) {
    AsyncPlan p{};
    p.tiles_m = (g.M + kTile - 1) / kTile;
    p.tiles_n = (g.N + kTile - 1) / kTile;
    const int tiles = p.tiles_m * p.tiles_n;
    const int nk = (g.K + kKT - 1) / kKT;
    int S = 1;
    const int cus = 256;  // one workgroup per CU; MI355X has 256 CUs
    if (tiles < cus) S = max(1, min(min(cus / tiles, nk / 16), 64));
    const int per = (nk + S - 1) / S;
    p.k_chunk = per * kKT;
    p.splits = (g.K + p.k_chunk - 1) / p.k_chunk;
    p.a_bytes = g.a_dtype == SNN_U8 ? align_up((size_t)g.M * g.K * 2) : 0;
    p.b_bytes = g.b_dtype == SNN_U8 ? align_up((size_t)g.N * g.K * 2) : 0;
    p.part_bytes = p.splits > 1 ? align_up((size_t)p.splits * g.M * g.N * sizeof(float)) : 0;
    return p;
}

}  // namespace

bool gemm_async_applies(const GemmArgs &g) {
    if (!g.allow_split || !g.a_kc || !g.b_kc) return false;
    if (mfma_type(g.a_dtype, g.b_dtype) < 0) return false;
    if (g.K % 8 != 0 || g.K < 256 || g.M < kTile || g.N < kTile) return false;
    if (g.a_dtype != SNN_U8 && g.lda % 8 != 0) return false;
    if (g.b_dtype != SNN_U8 && g.ldb % 8 != 0) return false;
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
    int64_t lda = g.lda, ldb = g.ldb;
    if (p.a_bytes) {
        uint16_t *d = reinterpret_cast<uint16_t *>(w);
        const int64_t n = (int64_t)g.M * (g.K / 8);
        if (mt == MT_F16)
            widen_kernel<MT_F16><<<blocks(n), kThreads, 0, s>>>(g.M, g.K, reinterpret_cast<const uint8_t *>(g.A), g.lda, d);
        else
            widen_kernel<MT_BF16><<<blocks(n), kThreads, 0, s>>>(g.M, g.K, reinterpret_cast<const uint8_t *>(g.A), g.lda, d);
        A = d;
        lda = g.K;
    }
    if (p.b_bytes) {
        uint16_t *d = reinterpret_cast<uint16_t *>(w + p.a_bytes);
        const int64_t n = (int64_t)g.N * (g.K / 8);
        if (mt == MT_F16)
            widen_kernel<MT_F16><<<blocks(n), kThreads, 0, s>>>(g.N, g.K, reinterpret_cast<const uint8_t *>(g.B), g.ldb, d);
        else
            widen_kernel<MT_BF16><<<blocks(n), kThreads, 0, s>>>(g.N, g.K, reinterpret_cast<const uint8_t *>(g.B), g.ldb, d);
        B = d;
        ldb = g.K;
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
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
    if (mt == MT_F16)
        gemm_async_kernel<MT_F16><<<grid, kThreads, 0, s>>>(g.M, g.N, g.K, p.k_chunk, p.tiles_n,
                                                            tiles, total, A, lda, B, ldb, out, ldo,
                                                            ss, bias, c_div);
    else
        gemm_async_kernel<MT_BF16><<<grid, kThreads, 0, s>>>(g.M, g.N, g.K, p.k_chunk, p.tiles_n,
                                                             tiles, total, A, lda, B, ldb, out, ldo,
                                                             ss, bias, c_div);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (p.splits > 1)
        e = launch_splitk_reduce(g.M, g.N, p.splits, out, g.C, g.ldc, g.bias, s, g.c_div);
    return e;
}

}  // namespace snn
