// Convolutional synapse of the paper's CSNN (Table I, "5C12-MP2-5C64-MP2"):
// a 5x5 valid cross-correlation, stride 1, plus bias, followed by 2x2 / 2
// max-pooling of the currents before the neuron.
//
// Both directions run as matrix products on the contraction kernels.  The
// conv outputs that some pool window reads are enumerated window by window:
//   row m = 4 q + d,  q = (nb * Hp + py) * Wp + px  (pooled cell),
//   d = 2 dy + dx     (position in the window, row-major),
// so conv output (oy, ox) = (2 py + dy, 2 px + dx), and a trailing odd row or
// column of conv outputs, which no window reads, is never computed.  With
// k = (c * 5 + ky) * 5 + kx (the weight layout [Co][Ci][5][5] flattened) and
// Kc = Ci * 25:
//
// Forward
//   col[m][k]  = x[nb, c, oy + ky, ox + kx]               (gather)
//   C[m][co]   = sum_k col[m][k] w[co][k] + bias[co]       (contraction)
//   cur[nb, co, py, px] = max_d C[4q + d][co], the first maximum in window
//                order; its d (0..3) is saved for the backward  (pool; the
//                16-bit contraction does it in its epilogue when it makes one
//                pass over K, a window being four rows of one lane's tile)
// At most four input channels (the input layer): conv1_pool_kernel computes
// the pooled currents directly.
//
// Backward, given dI = dL/dcur:
//   dC^T[co][m] = dI[nb, co, py, px] if d is the saved choice, else 0
//   dW[co][k]   = sum_m dC^T[co][m] col^T[k][m]           (contraction)
//   dx^T[k][m]  = sum_co w[co][k] dC^T[co][m]             (contraction)
//   dx[nb, c, y, x] = sum_{ky, kx} dx^T[(c, ky, kx)][m(nb, y - ky, x - kx)]
//                over the window rows that exist, in the fixed order ky, kx
//
// The contractions are the library's GEMMs (exact multi-part bf16 products
// with fp32 accumulation on the 16-bit matrix cores where they apply, fp32
// MFMA otherwise), so every sum is deterministic.  Where one image's window
// rows fit a workgroup (the CSNN's second layer: at most 16 pooled cells per
// channel, Ci * 25 <= 320, Co <= 64), each direction is one kernel that takes
// an image at a time with its tiles in LDS and registers: conv_fwd_kernel
// (contraction and pool, spike input), conv_dw_kernel (spike input) and
// conv_dx_kernel; col, C, dC^T and dx^T never reach HBM (see there).  Spikes are staged as
// bytes; an fp32 dC^T is written directly as three exact bf16 planes when the
// weight gradient runs on the 16-bit cores.  The bias gradient comes from the
// neuron scan's per-column sums.
#include "snn_internal.hpp"

namespace snn {
namespace {

constexpr int kThreads = 256;
constexpr int KS = 5;  // kernel size

// Sizes of the conv-as-GEMM buffers
struct ConvDims {
    int64_t Q;    // pooled cells, NB * Hp * Wp
    int64_t Mw;   // GEMM rows, 4 Q
    int Kc;       // Ci * 25
    int64_t ldk;  // row stride of col (elements), Kc rounded up to 16
    int64_t ldm;  // row stride of the transposed buffers (elements), Mw rounded up to 16
};

ConvDims dims_of(const ConvGeom &g) {
    ConvDims v{};
    v.Q = (int64_t)g.NB * g.Hp * g.Wp;
    v.Mw = 4 * v.Q;
    v.Kc = g.Ci * KS * KS;
    v.ldk = (v.Kc + 15) / 16 * 16;
    v.ldm = (v.Mw + 15) / 16 * 16;
    return v;
}

// 16 bytes of T, built element by element
template <typename T>
struct Chunk {
    static constexpr int N = 16 / (int)sizeof(T);
    union {
        T e[N];
        uint4 v;
    };
};

// Every conv tensor and GEMM buffer of a layer holds fewer than 2^31
// elements (checked when the layer is validated), so the kernels index in
// 32-bit integers.

// col[m][k0 .. k0 + N): one thread per 16-byte chunk of a row; k >= Kc is 0.
template <typename T>
__global__ __launch_bounds__(kThreads) void im2col_kernel(int Mw, int Kc, int ldk, int Ci, int H,
                                                          int W, int Hp, int Wp,
                                                          const T *__restrict__ x,
                                                          T *__restrict__ col) {
    constexpr int N = Chunk<T>::N;
    const int cpr = ldk / N;  // chunks per row
    const int idx = blockIdx.x * kThreads + threadIdx.x;
    if (idx >= Mw * cpr) return;
    const int m = idx / cpr, k0 = (idx - m * cpr) * N;
    const int q = m >> 2, d = m & 3, hw = Hp * Wp;
    const int nb = q / hw, p = q - nb * hw;
    const int py = p / Wp, px = p - py * Wp;
    const int base = (nb * Ci * H + 2 * py + (d >> 1)) * W + 2 * px + (d & 1);
    Chunk<T> ch;
#pragma unroll
    for (int i = 0; i < N; ++i) {
        const int k = min(k0 + i, Kc - 1);  // padding columns load a valid element, stored as 0
        const int c = k / (KS * KS), t = k - c * KS * KS, ky = t / KS, kx = t - ky * KS;
        const T e = x[base + (c * H + ky) * W + kx];
        ch.e[i] = (k0 + i < Kc) ? e : T(0);
    }
    *reinterpret_cast<uint4 *>(col + m * ldk + k0) = ch.v;
}

// The same gather with a workgroup per image: the image and a table of the
// x offsets of every k ((c * H + ky) * W + kx) are staged in LDS, so an
// element costs a table read, an add and an LDS read instead of the
// divisions that decompose k (and a global load).  For images of at most
// 16 KiB and Kc <= 1024.
constexpr int kIm2colLdsBytes = 16384;
constexpr int kIm2colMaxK = 1024;

template <typename T>
__global__ __launch_bounds__(kThreads) void im2col_lds_kernel(int Kc, int ldk, int Ci, int H, int W,
                                                              int Hp, int Wp, const T *__restrict__ x,
                                                              T *__restrict__ col) {
    constexpr int N = Chunk<T>::N;
    __shared__ __attribute__((aligned(16))) T xs[kIm2colLdsBytes / sizeof(T)];
    __shared__ __attribute__((aligned(16))) uint16_t off[kIm2colMaxK];
    const int img = Ci * H * W;
    const T *xi = x + (int64_t)blockIdx.x * img;
    for (int i = threadIdx.x; i < img; i += kThreads) xs[i] = xi[i];
    for (int k = threadIdx.x; k < ldk; k += kThreads) {
        const int kk = min(k, Kc - 1);  // padding columns read a valid element, stored as 0
        const int c = kk / (KS * KS), t = kk - c * KS * KS, ky = t / KS, kx = t - ky * KS;
        off[k] = (uint16_t)((c * H + ky) * W + kx);
    }
    __syncthreads();
    const int rows = 4 * Hp * Wp, cpr = ldk / N;
    T *colb = col + (int64_t)blockIdx.x * rows * ldk;
    for (int idx = threadIdx.x; idx < rows * cpr; idx += kThreads) {
        const int r = idx / cpr, k0 = (idx - r * cpr) * N;
        const int q = r >> 2, d = r & 3, py = q / Wp, px = q - py * Wp;
        const int base = (2 * py + (d >> 1)) * W + 2 * px + (d & 1);
        uint16_t o[N];
#pragma unroll
        for (int h = 0; h < N / 4; ++h) {
            const uint2 v = *reinterpret_cast<const uint2 *>(off + k0 + 4 * h);
            o[4 * h] = (uint16_t)(v.x & 0xffffu); o[4 * h + 1] = (uint16_t)(v.x >> 16);
            o[4 * h + 2] = (uint16_t)(v.y & 0xffffu); o[4 * h + 3] = (uint16_t)(v.y >> 16);
        }
        Chunk<T> ch;
#pragma unroll
        for (int i = 0; i < N; ++i) {
            const T e = xs[base + o[i]];
            ch.e[i] = (k0 + i < Kc) ? e : T(0);
        }
        *reinterpret_cast<uint4 *>(colb + (int64_t)r * ldk + k0) = ch.v;
    }
}

// col^T[k][m0 .. m0 + N): one thread per 16-byte chunk, N/4 whole windows
// (their four positions are x offsets 0, 1, W, W + 1); m >= Mw is 0.
template <typename T>
__global__ __launch_bounds__(kThreads) void im2col_t_kernel(int Mw, int Kc, int ldm, int Ci, int H,
                                                            int W, int Hp, int Wp,
                                                            const T *__restrict__ x,
                                                            T *__restrict__ colt) {
    constexpr int N = Chunk<T>::N;
    const int cpr = ldm / N;
    const int idx = blockIdx.x * kThreads + threadIdx.x;
    if (idx >= Kc * cpr) return;
    const int k = idx / cpr, m0 = (idx - k * cpr) * N;
    const int c = k / (KS * KS), t = k - c * KS * KS, ky = t / KS, kx = t - ky * KS;
    const int off = (c * H + ky) * W + kx;
    const int hw = Hp * Wp;
    Chunk<T> ch;
#pragma unroll
    for (int j = 0; j < N / 4; ++j) {
        const int qj = (m0 >> 2) + j;
        const int q = min(qj, (Mw >> 2) - 1);  // windows past the end load the last, stored as 0
        const int nb = q / hw, p = q - nb * hw, py = p / Wp, px = p - py * Wp;
        const T *xp = x + (nb * Ci * H + 2 * py) * W + 2 * px + off;
        const bool in = 4 * qj < Mw;
        const T v0 = xp[0], v1 = xp[1], v2 = xp[W], v3 = xp[W + 1];
        ch.e[4 * j] = in ? v0 : T(0);
        ch.e[4 * j + 1] = in ? v1 : T(0);
        ch.e[4 * j + 2] = in ? v2 : T(0);
        ch.e[4 * j + 3] = in ? v3 : T(0);
    }
    *reinterpret_cast<uint4 *>(colt + k * ldm + m0) = ch.v;
}

// Pool: a block takes QB consecutive pooled cells, stages their 4 * QB rows
// of C in LDS as [d][cell][co] (odd cell stride: the reads below are free of
// bank conflicts), then writes cur and the selection in output order
// (cell fastest, so consecutive lanes write consecutive addresses).
constexpr int kPoolLdsFloats = 8192;  // 32 KiB

__global__ __launch_bounds__(kThreads) void pool_kernel(int Q, int Co, int HW, int QB,
                                                        const float *__restrict__ C,
                                                        float *__restrict__ cur,
                                                        uint8_t *__restrict__ arg) {
    __shared__ float lds[kPoolLdsFloats];
    const int S = Co | 1;  // cell stride in LDS, odd
    const int q0 = blockIdx.x * QB;
    const int nq = min(QB, Q - q0);
    const float *Cb = C + q0 * 4 * Co;
    const int ne = nq * 4 * Co;  // <= kPoolLdsFloats
    constexpr int kPer = kPoolLdsFloats / kThreads;
    float v[kPer];
#pragma unroll
    for (int j = 0; j < kPer; ++j) {  // all loads in flight before the LDS stores
        const int e = threadIdx.x + j * kThreads;
        v[j] = e < ne ? Cb[e] : 0.f;
    }
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
        const int e = threadIdx.x + j * kThreads;
        if (e < ne) {
            const int row = e / Co, co = e - row * Co;
            lds[((row & 3) * QB + (row >> 2)) * S + co] = v[j];
        }
    }
    __syncthreads();
    const int no = nq * Co;
    for (int i = threadIdx.x; i < no; i += kThreads) {
        const int co = i / nq, qq = i - co * nq;
        float best = lds[qq * S + co];
        int a = 0;
#pragma unroll
        for (int d = 1; d < 4; ++d) {
            const float v = lds[(d * QB + qq) * S + co];
            if (v > best) {
                best = v;
                a = d;
            }
        }
        const int q = q0 + qq, nb = q / HW;
        const int o = (nb * Co + co) * HW + (q - nb * HW);
        cur[o] = best;
        arg[o] = (uint8_t)a;
    }
}

// At most four input channels (the input layer): the convolution and the pool
// in one kernel, without the gathered matrix or the unpooled currents.  A
// workgroup per image stages the image (as fp32) and the weights in LDS; a
// thread takes pooled currents (co, py, px), pooled column fastest, holds the
// 6x6 input patch of the window of one channel at a time in registers and
// accumulates the window's four conv outputs tap by tap (c, ky, kx ascending)
// with fp32 fma, then adds the bias and keeps the first maximum in window
// order, as the pool after the contraction.
constexpr int kDirectMaxHW = 4096;  // image pixels (all channels) staged in LDS
constexpr int kDirectMaxCo = 128;
constexpr int kDirectMaxCi = 4;    // 56 KiB of padded weights at most

bool direct_conv(const ConvGeom &g) {
    return g.Ci <= kDirectMaxCi && g.Ci * g.H * g.W <= kDirectMaxHW && g.Co <= kDirectMaxCo;
}

template <typename T, int CIM>  // CIM: most input channels (1, or up to kDirectMaxCi)
__global__ __launch_bounds__(kThreads) void conv1_pool_kernel(int Ci, int H, int W, int Co, int Hp,
                                                              int Wp, const T *__restrict__ x,
                                                              const float *__restrict__ w,
                                                              const float *__restrict__ bias,
                                                              float *__restrict__ cur,
                                                              uint8_t *__restrict__ arg) {
    constexpr int WS = 28;  // weights of one (output, input) channel pair, padded to 16 bytes
    __shared__ __attribute__((aligned(16))) float xs[kDirectMaxHW];
    __shared__ __attribute__((aligned(16))) float wsh[kDirectMaxCo * CIM * WS];
    const int64_t nb = blockIdx.x;
    const int hw = H * W;
    const T *xi = x + nb * Ci * hw;
    for (int i = threadIdx.x; i < Ci * hw; i += kThreads) xs[i] = (float)xi[i];
    for (int i = threadIdx.x; i < Co * Ci * WS; i += kThreads) {
        const int cc = i / WS, t = i - cc * WS;  // cc = co * Ci + c
        wsh[i] = t < KS * KS ? w[cc * KS * KS + t] : 0.f;
    }
    __syncthreads();
    const bool pairs = (W & 1) == 0;  // patch rows start at even offsets: 8-byte reads
    const int cells = Hp * Wp, total = Co * cells;
    float *cb = cur + nb * total;
    uint8_t *ab = arg + nb * total;
    for (int o = threadIdx.x; o < total; o += kThreads) {
        const int co = o / cells, p = o - co * cells;
        const int py = p / Wp, px = p - py * Wp;
        float acc[4] = {0.f, 0.f, 0.f, 0.f};
        for (int ci = 0; ci < (CIM == 1 ? 1 : Ci); ++ci) {  // k = (ci, ky, kx) ascending
            const float *xp = xs + ci * hw + 2 * py * W + 2 * px;
            float patch[KS + 1][KS + 1];
            if (pairs) {
#pragma unroll
                for (int r = 0; r <= KS; ++r)
#pragma unroll
                    for (int c = 0; c <= KS; c += 2) {
                        const float2 v = *reinterpret_cast<const float2 *>(xp + r * W + c);
                        patch[r][c] = v.x;
                        patch[r][c + 1] = v.y;
                    }
            } else {
#pragma unroll
                for (int r = 0; r <= KS; ++r)
#pragma unroll
                    for (int c = 0; c <= KS; ++c) patch[r][c] = xp[r * W + c];
            }
            float wv[WS];
#pragma unroll
            for (int q = 0; q < WS / 4; ++q) {
                const float4 v = *reinterpret_cast<const float4 *>(wsh + (co * Ci + ci) * WS + 4 * q);
                wv[4 * q] = v.x; wv[4 * q + 1] = v.y; wv[4 * q + 2] = v.z; wv[4 * q + 3] = v.w;
            }
#pragma unroll
            for (int ky = 0; ky < KS; ++ky)
#pragma unroll
                for (int kx = 0; kx < KS; ++kx) {
                    const float wv1 = wv[ky * KS + kx];
#pragma unroll
                    for (int d = 0; d < 4; ++d)
                        acc[d] = __builtin_fmaf(patch[(d >> 1) + ky][(d & 1) + kx], wv1, acc[d]);
                }
        }
        const float bco = bias ? bias[co] : 0.f;
        float best = acc[0] + bco;
        int a = 0;
#pragma unroll
        for (int d = 1; d < 4; ++d) {
            const float v = acc[d] + bco;
            if (v > best) {
                best = v;
                a = d;
            }
        }
        cb[o] = best;
        ab[o] = (uint8_t)a;
    }
}

__device__ inline uint32_t bf16_rne(float x) {
    const uint32_t b = __float_as_uint(x);
    return (b + 0x7fffu + ((b >> 16) & 1u)) >> 16;
}

// dC^T[co][4q .. 4q + 3] from the pooled gradient and the saved choice
// (unless `dct` is null); with `planes`, also its three exact bf16 parts
// (hi, mid, lo), planes Co * ldm elements apart.
__global__ __launch_bounds__(kThreads) void unpool_t_kernel(int Q, int Co, int HW, int ldm,
                                                            const float *__restrict__ dI,
                                                            const uint8_t *__restrict__ arg,
                                                            float *__restrict__ dct,
                                                            uint16_t *__restrict__ planes) {
    const int idx = blockIdx.x * kThreads + threadIdx.x;
    if (idx >= Q * Co) return;
    const int co = idx / Q, q = idx - co * Q;
    const int nb = q / HW;
    const int src = (nb * Co + co) * HW + (q - nb * HW);
    const float g = dI[src];
    const int a = arg[src];
    float v[4];
#pragma unroll
    for (int d = 0; d < 4; ++d) v[d] = (d == a) ? g : 0.f;
    const int o = co * ldm + 4 * q;
    if (dct) *reinterpret_cast<float4 *>(dct + o) = make_float4(v[0], v[1], v[2], v[3]);
    if (planes) {
        uint32_t p[3][4];
#pragma unroll
        for (int d = 0; d < 4; ++d) {
            const uint32_t hi = bf16_rne(v[d]);
            const float r = v[d] - __uint_as_float(hi << 16);
            const uint32_t mid = bf16_rne(r);
            p[0][d] = hi;
            p[1][d] = mid;
            p[2][d] = bf16_rne(r - __uint_as_float(mid << 16));
        }
        const int64_t ps = (int64_t)Co * ldm;
#pragma unroll
        for (int k = 0; k < 3; ++k)
            *reinterpret_cast<uint2 *>(planes + k * ps + o) =
                make_uint2(p[k][0] | (p[k][1] << 16), p[k][2] | (p[k][3] << 16));
    }
}

// dx[nb, c, y, x] = sum over (ky, kx) of dx^T[(c, ky, kx)][m(nb, y - ky, x - kx)]
// for the conv outputs some window reads; fixed order ky, kx.  Lanes take the
// input pixels in 2x2 blocks, (y, x) = (2 py + dy, 2 px + dx) with (dy, dx)
// fastest, the order of the window rows m: for each (ky, kx) a wave then reads
// one or two contiguous runs of dx^T.
__global__ __launch_bounds__(kThreads) void col2im_kernel(int total, int Ci, int H, int W, int PH,
                                                          int PW, int Hp, int Wp, int ldm,
                                                          const float *__restrict__ dxt,
                                                          float *__restrict__ dx) {
    const int idx = blockIdx.x * kThreads + threadIdx.x;
    if (idx >= total) return;
    const int e = idx & 3, cell = idx >> 2;
    const int r = cell / PW, px = cell - r * PW;
    const int img = r / PH, py = r - img * PH;
    const int yy = 2 * py + (e >> 1), xx = 2 * px + (e & 1);
    if (yy >= H || xx >= W) return;
    const int nb = img / Ci, c = img - nb * Ci;
    // all 25 loads are issued unconditionally (a tap outside the windows
    // reads row 0 of its k and is not added), so they overlap in flight
    float v[KS * KS];
    bool ok[KS * KS];
#pragma unroll
    for (int ky = 0; ky < KS; ++ky) {
        const int oy = yy - ky;
        const bool oky = oy >= 0 && oy < 2 * Hp;
        const int mrow = (nb * Hp + (oy >> 1)) * Wp;
#pragma unroll
        for (int kx = 0; kx < KS; ++kx) {
            const int ox = xx - kx;
            const bool okx = ox >= 0 && ox < 2 * Wp;
            const int m = (oky && okx) ? (mrow + (ox >> 1)) * 4 + 2 * (oy & 1) + (ox & 1) : 0;
            v[ky * KS + kx] = dxt[((c * KS + ky) * KS + kx) * ldm + m];
            ok[ky * KS + kx] = oky && okx;
        }
    }
    float acc = 0.f;
#pragma unroll
    for (int t = 0; t < KS * KS; ++t)
        if (ok[t]) acc += v[t];
    dx[(img * H + yy) * W + xx] = acc;
}

// ---- input gradient in one pass ----------------------------------------------
// When one image's product fits a workgroup (Ci * 25 <= 320, Co <= 64, at most
// 16 pooled cells per channel, so at most 64 window rows), dx^T never reaches
// HBM.  A workgroup takes one image at a time:
//   dcol[m][k] = sum_co dC[m][co] w[co][k]      (16 x 16 x 32 bf16 MFMA tiles)
// with dC[m][co] = dI[co][q] if the saved choice of (co, q) is d (m = 4 q + d),
// else 0; dcol goes to LDS as [k][m], and dx is gathered from it as
// col2im_kernel does (fixed order ky, kx over the window rows that exist).
// The weights stay in registers for the whole launch as three exact bf16
// parts (hi, mid, lo); dC is staged in LDS split the same way, and six of the
// nine part products are summed, the smallest first.  The three left out
// (mid lo, lo mid, lo lo) are below 2^-26 of |dC w| (|mid| <= 2^-9 |x|,
// |lo| <= 2^-18 |x|), a quarter of an fp32 rounding, so every product is
// fp32-accurate before the fp32 accumulation.  Eight waves: wave v takes
// every row tile and the column tiles v, v + 8, v + 16.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kDxThreads = 512;
constexpr int kDxMaxK = 320;                  // Ci * 25: 20 column tiles
constexpr int kDxTileRows = 24 * 16;          // dcol^T rows the eight waves store
constexpr int kDxMaxCo = 64;                  // two k-steps of 32
constexpr int kDxMaxCells = 16;               // pooled cells per channel
constexpr int kDxRows = 4 * kDxMaxCells;      // window rows: four row tiles
constexpr int kDxLdm = kDxRows + 4;           // dcol^T row stride (floats): the
                                              // 16-byte stores of 16 lanes, k
                                              // apart, hit distinct bank groups
constexpr int kDxLdc = kDxMaxCo + 8;          // dC part row stride (bf16): the
                                              // 16-byte reads of 16 lanes, m
                                              // apart, hit distinct bank groups
constexpr int kDxPer = kDxMaxCo * kDxMaxCells / kDxThreads;  // (co, q) per thread

// A workgroup barrier that waits for the wave's LDS accesses only: the loads
// of the next image and the stores of dx stay in flight across it (nothing
// in this kernel reads global memory that another wave writes).
__device__ inline void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

__device__ inline floatx4 mfma_bf16(const u32x4 &a, const u32x4 &b, const floatx4 &c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

template <int G>
__global__ __launch_bounds__(kDxThreads) void conv_dx_kernel(
    int NB, int Ci, int H, int W, int Co, int Hp, int Wp, const float *__restrict__ dI,
    const uint8_t *__restrict__ arg, const float *__restrict__ w, float *__restrict__ dx) {
    __shared__ __attribute__((aligned(16))) float dcol[kDxTileRows * kDxLdm];
    __shared__ __attribute__((aligned(16))) uint16_t dcp[2][3][kDxRows * kDxLdc];
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int col = lane & 15, kg = lane >> 4;
    const int HW = Hp * Wp, Kc = Ci * KS * KS, CHW = Co * HW;
    const bool two_k = Co > 32;

    // rows past 4 HW and columns past Co stay zero for the whole launch, and
    // so do the padding columns m = 64..67 of dcol^T, which the gather reads
    // for a tap outside the windows
    for (int i = tid; i < 2 * 3 * kDxRows * kDxLdc / 2; i += kDxThreads)
        reinterpret_cast<uint32_t *>(&dcp[0][0][0])[i] = 0u;
    for (int i = tid; i < kDxTileRows * (kDxLdm - kDxRows); i += kDxThreads)
        dcol[(i >> 2) * kDxLdm + kDxRows + (i & 3)] = 0.f;

    // Gather: thread (cg, p) < (G, H * W) takes pixel p of channels cg + G j.
    // Its 25 taps read dcol^T[(c * 25 + t)][m_t] for the window row m_t under
    // the tap, or the zero padding; tap[t] holds the offset for c = cg.
    const int HWi = H * W, npix = Ci * HWi;
    const bool gact = tid < G * HWi;
    const int cg = gact ? tid / HWi : 0, pix = gact ? tid - cg * HWi : 0;
    int tap[KS * KS];
    {
        const int y = pix / W, xx = pix - (pix / W) * W;
#pragma unroll
        for (int ky = 0; ky < KS; ++ky)
#pragma unroll
            for (int kx = 0; kx < KS; ++kx) {
                const int oy = y - ky, ox = xx - kx;
                const bool ok = oy >= 0 && oy < 2 * Hp && ox >= 0 && ox < 2 * Wp;
                const int m = ok ? 4 * ((oy >> 1) * Wp + (ox >> 1)) + 2 * (oy & 1) + (ox & 1)
                                 : kDxRows;
                tap[ky * KS + kx] = (cg * KS * KS + ky * KS + kx) * kDxLdm + m;
            }
    }

    // B fragments of the weights: lane (col, kg) holds w[32 ks + 8 kg + e][16 nt + col]
    // (zero past Kc and Co: the tiles there multiply zeros)
    u32x4 bw[3][2][3];
#pragma unroll
    for (int j = 0; j < 3; ++j)
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            const int n = (wv + 8 * j) * 16 + col;
            uint32_t h[3][8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int co = ks * 32 + 8 * kg + e;
                const float x = (n < Kc && co < Co) ? w[co * Kc + n] : 0.f;
                h[0][e] = bf16_rne(x);
                const float r = x - __uint_as_float(h[0][e] << 16);
                h[1][e] = bf16_rne(r);
                h[2][e] = bf16_rne(r - __uint_as_float(h[1][e] << 16));
            }
#pragma unroll
            for (int p = 0; p < 3; ++p)
                bw[j][ks][p] = u32x4{h[p][0] | (h[p][1] << 16), h[p][2] | (h[p][3] << 16),
                                     h[p][4] | (h[p][5] << 16), h[p][6] | (h[p][7] << 16)};
        }

    float gnext[kDxPer];
    int anext[kDxPer];
    // Loads and LDS stores without branches (clamped addresses; a thread past
    // the image writes a padding column), so the wait for the loaded values
    // sits at their one use on every path and covers nothing issued later.
    auto fetch = [&](int nb) {
#pragma unroll
        for (int r = 0; r < kDxPer; ++r) {
            const int i = tid + r * kDxThreads;
            const bool in = nb < NB && i < CHW;
            const int o = min(nb, NB - 1) * CHW + min(i, CHW - 1);
            const float g = dI[o];
            const int a = arg[o];
            gnext[r] = in ? g : 0.f;
            anext[r] = in ? a : 0;
        }
    };
    // dC of an image as three bf16 parts, [part][m][co]
    auto stage = [&](uint16_t (*dst)[kDxRows * kDxLdc]) {
#pragma unroll
        for (int r = 0; r < kDxPer; ++r) {
            const int i = tid + r * kDxThreads;
            const float g = gnext[r];
            const int a = anext[r];
            const uint32_t hi = bf16_rne(g);
            const float rr = g - __uint_as_float(hi << 16);
            const uint32_t mid = bf16_rne(rr);
            const uint32_t lo = bf16_rne(rr - __uint_as_float(mid << 16));
            const bool in = i < CHW;
            const int co = i / HW, q = i - co * HW;
#pragma unroll
            for (int d = 0; d < 4; ++d) {
                const bool on = a == d;
                const int o = in ? (4 * q + d) * kDxLdc + co : kDxMaxCo;  // padding of row 0
                dst[0][o] = on ? (uint16_t)hi : (uint16_t)0;
                dst[1][o] = on ? (uint16_t)mid : (uint16_t)0;
                dst[2][o] = on ? (uint16_t)lo : (uint16_t)0;
            }
        }
    };

    // Per image n: products from dcp[n & 1]; barrier (the gather of n - 1 is
    // done with dcol); dcol stored; image n + 1 staged into the other buffer;
    // barrier; gather.  The loads of n + 1 are issued before the products of
    // n and the stores of dx drain under the next products, so no wait for
    // global memory lands between two barriers.
    fetch(blockIdx.x);
    lds_barrier();  // the zeroed buffers
    stage(dcp[0]);
    lds_barrier();
    int buf = 0;
    for (int nb = blockIdx.x; nb < NB; nb += gridDim.x, buf ^= 1) {
        fetch(nb + gridDim.x);

        floatx4 acc[4][3];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 3; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
        const uint16_t(*src)[kDxRows * kDxLdc] = dcp[buf];
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            if (ks == 1 && !two_k) break;
            // A fragments: lane (col, kg) holds dC[16 mt + col][32 ks + 8 kg + e]
            u32x4 ap[4][3];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int p = 0; p < 3; ++p)
                    ap[i][p] = *reinterpret_cast<const u32x4 *>(
                        &src[p][(16 * i + col) * kDxLdc + 32 * ks + 8 * kg]);
            // part products smallest first (mid mid, lo hi, hi lo, mid hi, hi mid,
            // hi hi); the twelve tiles interleave
            constexpr int pa[6] = {1, 2, 0, 1, 0, 0}, pb[6] = {1, 0, 2, 0, 1, 0};
#pragma unroll
            for (int t = 0; t < 6; ++t)
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int j = 0; j < 3; ++j)
                        acc[i][j] = mfma_bf16(ap[i][pa[t]], bw[j][ks][pb[t]], acc[i][j]);
        }
        lds_barrier();  // the gather of the previous image is done with dcol
        // D fragment: lane (col, kg) holds dcol[16 mt + 4 kg + r][16 nt + col], r = 0..3,
        // stored as dcol^T[k][m], four consecutive m in one 16-byte store
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 3; ++j)
                *reinterpret_cast<floatx4 *>(dcol + ((wv + 8 * j) * 16 + col) * kDxLdm + 16 * i +
                                             4 * kg) = acc[i][j];
        stage(dcp[buf ^ 1]);
        lds_barrier();
        // fixed order t = 5 ky + kx; a tap outside the windows adds the zero padding
        if (gact) {
            float *dxi = dx + (int64_t)nb * npix + pix;
#pragma unroll
            for (int j = 0; j < (kDxMaxK / (KS * KS) + G - 1) / G; ++j) {
                const int c = cg + G * j;
                if (c >= Ci) break;
                const float *dc = dcol + G * j * KS * KS * kDxLdm;
                float v[KS * KS];
#pragma unroll
                for (int t = 0; t < KS * KS; ++t) v[t] = dc[tap[t]];
                float acc = 0.f;
#pragma unroll
                for (int t = 0; t < KS * KS; ++t) acc += v[t];
                dxi[c * HWi] = acc;
            }
        }
    }
}

// ---- weight gradient in one pass ---------------------------------------------
// For the same layers up to 32 pooled cells per channel (128 window rows), on
// spike images of whole 4-byte words: a workgroup takes one image at a time
// and accumulates, over all its images,
//   dW[co][k] = sum_m dC^T[co][m] col[m][k]       (16 x 16 x 32 bf16 MFMA tiles)
// with dC^T staged in LDS as three exact bf16 parts ([part][co][m]: four
// window rows of a pooled cell are one 8-byte store) and col[m][k] read
// straight from the image, staged in LDS as bf16 0 / 1: lane (n, g) of a
// B fragment takes the 8 window rows 32 s + 8 g .. + 7, two pooled cells of
// four positions (x offsets 0, 1, W, W + 1 from the cell's corner under tap
// k).  The three part products per tile are exact and summed smallest first
// in fp32; each workgroup writes its partial sums, which splitk_reduce adds
// in a fixed order.  Eight waves: wave v takes every output-channel tile and
// the k tiles v, v + 8, v + 16.  The image and the parts of the next image
// are loaded during the products (two images ahead) and staged after a
// barrier.
constexpr int kDwMaxGrid = 256;                   // partial sums written
constexpr int kFwMaxCells = 32;                   // pooled cells per channel for the
                                                  // forward and the weight gradient
constexpr int kFwRows = 4 * kFwMaxCells;          // window rows: up to 8 row tiles
constexpr int kDwLdm = kFwRows + 8;               // dC^T part row stride (bf16): 272-byte
                                                  // rows, so the 16-byte reads of 16
                                                  // lanes, co apart, hit distinct
                                                  // bank groups
constexpr int kDwMaxX = kDxMaxK / (KS * KS) * kDxThreads;  // image elements staged
constexpr int kDwXPer = kDwMaxX / 4 / kDxThreads; // 4-byte image words loaded per thread
constexpr int kDwPer = kDxMaxCo * kFwMaxCells / kDxThreads;  // (co, q) per thread

// bf16 of four spike bytes (every byte value is exact), as two words
__device__ inline uint2 bytes4_bf16(uint32_t w) {
    uint32_t h[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) h[e] = __float_as_uint((float)((w >> (8 * e)) & 0xffu)) >> 16;
    return make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16));
}

__global__ __launch_bounds__(kDxThreads) void conv_dw_kernel(
    int NB, int Ci, int H, int W, int Co, int Hp, int Wp, const float *__restrict__ dI,
    const uint8_t *__restrict__ arg, const uint8_t *__restrict__ x, float *__restrict__ partial) {
    __shared__ __attribute__((aligned(16))) uint16_t dct[3][kDxMaxCo * kDwLdm];
    __shared__ __attribute__((aligned(16))) uint16_t xs[kDwMaxX];
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int col = lane & 15, kg = lane >> 4;
    const int HW = Hp * Wp, Kc = Ci * KS * KS, CHW = Co * HW, HWi = H * W, npx = Ci * HWi;
    const int nxw = npx / 4;  // image words (npx is a multiple of 4)
    const int nms = (4 * HW + 31) / 32;  // 32-row steps of the window rows

    // window rows past 4 HW and channels past Co stay zero for the whole launch
    for (int i = tid; i < 3 * kDxMaxCo * kDwLdm / 2; i += kDxThreads)
        reinterpret_cast<uint32_t *>(&dct[0][0])[i] = 0u;

    // per lane: the image offset of its k under each of its k tiles (k past Kc
    // reads a valid element; those output columns are not stored), and the
    // corner of its two pooled cells per 32 window rows (cells past HW read
    // element 0: their dC^T rows are zero)
    int koff[3], cb[kFwRows / 32][2];
#pragma unroll
    for (int j = 0; j < 3; ++j) {
        const int k = (wv + 8 * j) * 16 + col;
        const int c = k / (KS * KS), t = k - c * KS * KS, ky = t / KS, kx = t - ky * KS;
        koff[j] = k < Kc ? c * HWi + ky * W + kx : 0;
    }
#pragma unroll
    for (int ms = 0; ms < kFwRows / 32; ++ms)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int q = 8 * ms + 2 * kg + h, py = q / Wp, px = q - py * Wp;
            cb[ms][h] = q < HW ? 2 * py * W + 2 * px : 0;
        }

    // The loads of an image are issued two images ahead, into one of two
    // register sets, so a whole image's products hide their latency.
    struct Next {
        float g[kDwPer];
        int a[kDwPer];
        uint32_t x[kDwXPer];
    };
    auto fetch = [&](Next &n, int nb) {
        const int b = min(nb, NB - 1);
#pragma unroll
        for (int r = 0; r < kDwPer; ++r) {
            const int i = tid + r * kDxThreads;
            const int o = b * CHW + min(i, CHW - 1);
            const float g = dI[o];
            n.a[r] = arg[o];
            n.g[r] = (nb < NB && i < CHW) ? g : 0.f;
        }
        const uint32_t *xw = reinterpret_cast<const uint32_t *>(x) + (int64_t)b * nxw;
#pragma unroll
        for (int r = 0; r < kDwXPer; ++r) {
            const int i = tid + r * kDxThreads;
            if (r * kDxThreads < nxw) n.x[r] = xw[min(i, nxw - 1)];
        }
    };
    auto stage = [&](const Next &n) {
#pragma unroll
        for (int r = 0; r < kDwPer; ++r) {
            const int i = tid + r * kDxThreads;
            const float g = n.g[r];
            const uint32_t hi = bf16_rne(g);
            const float rr = g - __uint_as_float(hi << 16);
            const uint32_t mid = bf16_rne(rr);
            const uint32_t lo = bf16_rne(rr - __uint_as_float(mid << 16));
            const uint32_t pv[3] = {hi, mid, lo};
            if (i < CHW) {
                const int co = i / HW, q = i - co * HW, a = n.a[r];
#pragma unroll
                for (int pp = 0; pp < 3; ++pp) {
                    const uint32_t v = pv[pp];
                    const uint2 w2 = make_uint2((a == 0 ? v : 0u) | ((a == 1 ? v : 0u) << 16),
                                                (a == 2 ? v : 0u) | ((a == 3 ? v : 0u) << 16));
                    *reinterpret_cast<uint2 *>(&dct[pp][co * kDwLdm + 4 * q]) = w2;
                }
            }
        }
#pragma unroll
        for (int r = 0; r < kDwXPer; ++r) {
            const int i = tid + r * kDxThreads;
            if (r * kDxThreads < nxw && i < nxw)
                *reinterpret_cast<uint2 *>(&xs[4 * i]) = bytes4_bf16(n.x[r]);
        }
    };

    floatx4 acc[4][3];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 3; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
    auto products = [&]() {
#pragma unroll
        for (int ms = 0; ms < kFwRows / 32; ++ms) {
            if (ms < nms) {
                // A fragments, all parts: lane (col, kg) holds dC^T[16 ct + col][32 ms + 8 kg + e]
                u32x4 ap[3][4];
#pragma unroll
                for (int pp = 0; pp < 3; ++pp)
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        ap[pp][i] = *reinterpret_cast<const u32x4 *>(
                            &dct[pp][(16 * i + col) * kDwLdm + 32 * ms + 8 * kg]);
                // B fragments: lane (col, kg) holds col[32 ms + 8 kg + e][16 kt + col]
                u32x4 bx[3];
#pragma unroll
                for (int j = 0; j < 3; ++j) {
                    uint32_t h4[4];
#pragma unroll
                    for (int h = 0; h < 2; ++h) {
                        const uint16_t *q = xs + koff[j] + cb[ms][h];
                        h4[2 * h] = (uint32_t)q[0] | ((uint32_t)q[1] << 16);
                        h4[2 * h + 1] = (uint32_t)q[W] | ((uint32_t)q[W + 1] << 16);
                    }
                    bx[j] = u32x4{h4[0], h4[1], h4[2], h4[3]};
                }
                // parts smallest first
#pragma unroll
                for (int pp = 2; pp >= 0; --pp)
#pragma unroll
                    for (int i = 0; i < 4; ++i)
#pragma unroll
                        for (int j = 0; j < 3; ++j)
                            acc[i][j] = mfma_bf16(ap[pp][i], bx[j], acc[i][j]);
            }
        }
    };

    Next n0, n1;
    const int G = gridDim.x;
    int nb = blockIdx.x;
    fetch(n0, nb);
    fetch(n1, nb + G);
    lds_barrier();  // the zeroed parts
    stage(n0);
    lds_barrier();
    while (true) {
        fetch(n0, nb + 2 * G);
        products();
        lds_barrier();  // every wave is done with the parts and the image
        nb += G;
        if (nb >= NB) break;
        stage(n1);
        lds_barrier();
        fetch(n1, nb + 2 * G);
        products();
        lds_barrier();
        nb += G;
        if (nb >= NB) break;
        stage(n0);
        lds_barrier();
    }
    // D fragment: lane (col, kg) holds dW[16 ct + 4 kg + r][16 kt + col]
    float *out = partial + (int64_t)blockIdx.x * Co * Kc;
#pragma unroll
    for (int j = 0; j < 3; ++j) {
        const int k = (wv + 8 * j) * 16 + col;
        if (k >= Kc) continue;
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int co = 16 * i + 4 * kg + r;
                if (co < Co) out[co * Kc + k] = acc[i][j][r];
            }
    }
}

// ---- forward in one pass --------------------------------------------------------
// For the same layers as the weight gradient above (spike images of whole
// 4-byte words, up to 32 pooled cells), without col or C in HBM: a workgroup
// takes one image at a time, gathers col[m][k] for its window rows into LDS
// (bf16 0 / 1, from the image staged there), and computes
//   C[m][co] = sum_k col[m][k] w[co][k] + bias[co]  (16 x 16 x 32 bf16 MFMA tiles)
// with the weights held in registers as three exact bf16 parts: exact
// products, summed smallest part first in fp32.  The pool needs no exchange: the
// four window rows of a pooled cell are the four accumulator rows of one lane,
// so each lane adds the bias, keeps the first maximum and stores cur and the
// choice.  Eight waves: wave v takes row tiles (v & 1) + {0, 2} (+ {4, 6}
// past 16 pooled cells) and output channels 16 (v >> 1) .. + 15.
constexpr int kFwLdk = kDxMaxK + 8;  // col row stride (bf16): 656-byte rows, so the
                                     // 16-byte reads of 16 lanes, rows apart, hit
                                     // distinct bank groups
constexpr int kFwChunks = kDxMaxK / 8;  // 8-column chunks of col

template <int MPW>  // row tiles per wave: 2 (at most 16 pooled cells) or 4
__global__ __launch_bounds__(kDxThreads) void conv_fwd_kernel(
    int NB, int Ci, int H, int W, int Co, int Hp, int Wp, const uint8_t *__restrict__ x,
    const float *__restrict__ w, const float *__restrict__ bias, float *__restrict__ cur,
    uint8_t *__restrict__ arg) {
    constexpr int ROWS = 32 * MPW;
    __shared__ __attribute__((aligned(16))) uint16_t colb[ROWS * kFwLdk];
    __shared__ __attribute__((aligned(16))) uint16_t xs[2][kDwMaxX];
    __shared__ __attribute__((aligned(16))) int kot[kDxMaxK];  // image offset of column k
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int col = lane & 15, kg = lane >> 4;
    const int wvu = __builtin_amdgcn_readfirstlane(wv);  // uniform across the wave
    const int wm = wvu & 1, wn = wvu >> 1;
    const int HW = Hp * Wp, Kc = Ci * KS * KS, HWi = H * W, npx = Ci * HWi, Mi = 4 * HW;
    const int nxw = npx / 4;  // image words (npx is a multiple of 4)
    const int KT = (Kc + 31) / 32, MT = (Mi + 15) / 16;

    // B fragments: lane (col, kg) holds w[16 wn + col][32 ks + 8 kg + e] as three parts
    const int co = 16 * wn + col;
    u32x4 bw[kDxMaxK / 32][3];
#pragma unroll
    for (int ks = 0; ks < kDxMaxK / 32; ++ks) {
        uint32_t h[3][8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int k = ks * 32 + 8 * kg + e;
            const float v = (co < Co && k < Kc) ? w[co * Kc + k] : 0.f;
            h[0][e] = bf16_rne(v);
            const float r = v - __uint_as_float(h[0][e] << 16);
            h[1][e] = bf16_rne(r);
            h[2][e] = bf16_rne(r - __uint_as_float(h[1][e] << 16));
        }
#pragma unroll
        for (int pp = 0; pp < 3; ++pp)
            bw[ks][pp] = u32x4{h[pp][0] | (h[pp][1] << 16), h[pp][2] | (h[pp][3] << 16),
                               h[pp][4] | (h[pp][5] << 16), h[pp][6] | (h[pp][7] << 16)};
    }
    const float bco = (bias && co < Co) ? bias[co] : 0.f;

    // The gather: lane l of wave v writes rows m = l and l + 64 of col,
    // columns 8 ch .. + 7 for ch = v, v + 8, ..; the image offset of a row
    // (mo) is the lane's, that of a column (kot, read as a broadcast) is the
    // same for the whole wave.  Lanes, 64 window rows (16 pooled cells), read distinct words: no
    // bank conflicts.  A row past the windows reads the image corner (its
    // outputs are not stored); a column past Kc reads its channel's corner
    // (its weights are zero).
    const int wvs = wvu;
    for (int k = tid; k < kDxMaxK; k += kDxThreads) {
        const int c = k / (KS * KS), t = k - c * KS * KS, ky = t / KS, kx = t - ky * KS;
        kot[k] = k < Kc ? c * HWi + ky * W + kx : 0;
    }
    int mo[MPW / 2];
#pragma unroll
    for (int r = 0; r < MPW / 2; ++r) {
        const int m = lane + 64 * r, q = m >> 2, d = m & 3, py = q / Wp, px = q - py * Wp;
        mo[r] = m < Mi ? (2 * py + (d >> 1)) * W + 2 * px + (d & 1) : 0;
    }
    struct Next {
        uint32_t x[kDwXPer];
    };
    auto fetch = [&](Next &n, int nb) {
        const int b = min(nb, NB - 1);
        const uint32_t *xw = reinterpret_cast<const uint32_t *>(x) + (int64_t)b * nxw;
#pragma unroll
        for (int r = 0; r < kDwXPer; ++r) {
            const int i = tid + r * kDxThreads;
            if (r * kDxThreads < nxw) n.x[r] = xw[min(i, nxw - 1)];
        }
    };
    auto stage = [&](const Next &n, uint16_t *dst) {
#pragma unroll
        for (int r = 0; r < kDwXPer; ++r) {
            const int i = tid + r * kDxThreads;
            if (r * kDxThreads < nxw && i < nxw)
                *reinterpret_cast<uint2 *>(&dst[4 * i]) = bytes4_bf16(n.x[r]);
        }
    };
    auto build = [&](const uint16_t *src) {
#pragma unroll
        for (int j = 0; j < kFwChunks / 8; ++j) {
            const int ch = wvs + 8 * j;
            if (ch < 4 * KT) {
                const int4 k0 = *reinterpret_cast<const int4 *>(&kot[8 * ch]);
                const int4 k1 = *reinterpret_cast<const int4 *>(&kot[8 * ch + 4]);
                const int ko[8] = {k0.x, k0.y, k0.z, k0.w, k1.x, k1.y, k1.z, k1.w};
#pragma unroll
                for (int r = 0; r < MPW / 2; ++r) {
                    const int m = lane + 64 * r;
                    if (m < 16 * MT) {
                        uint32_t hv[8];
#pragma unroll
                        for (int e = 0; e < 8; ++e) hv[e] = src[mo[r] + ko[e]];
                        *reinterpret_cast<u32x4 *>(&colb[m * kFwLdk + 8 * ch]) =
                            u32x4{hv[0] | (hv[1] << 16), hv[2] | (hv[3] << 16),
                                  hv[4] | (hv[5] << 16), hv[6] | (hv[7] << 16)};
                    }
                }
            }
        }
    };

    // The registers hold the image after the one being multiplied: it is
    // staged into the other buffer during the products, and the loads of the
    // one after it are issued there.
    Next n;
    const int G = gridDim.x;
    int nb = blockIdx.x, buf = 0;
    fetch(n, nb);
    stage(n, xs[0]);
    fetch(n, nb + G);
    lds_barrier();
    while (true) {
        build(xs[buf]);
        lds_barrier();  // col complete
        // (the other buffer's last reader, the previous gather, finished
        // before the barrier above)
        stage(n, xs[buf ^ 1]);
        fetch(n, nb + 2 * G);
        floatx4 acc[MPW];
#pragma unroll
        for (int i = 0; i < MPW; ++i) acc[i] = floatx4{0.f, 0.f, 0.f, 0.f};
        // (tiles past the window rows multiply stale rows; they are not stored)
#pragma unroll
        for (int ks = 0; ks < kDxMaxK / 32; ++ks) {
            if (ks < KT) {
                u32x4 a[MPW];
#pragma unroll
                for (int i = 0; i < MPW; ++i)
                    a[i] = *reinterpret_cast<const u32x4 *>(
                        &colb[(16 * (wm + 2 * i) + col) * kFwLdk + 32 * ks + 8 * kg]);
#pragma unroll
                for (int pp = 2; pp >= 0; --pp)
#pragma unroll
                    for (int i = 0; i < MPW; ++i) acc[i] = mfma_bf16(a[i], bw[ks][pp], acc[i]);
            }
        }
        // pool: lane (col, kg) holds C rows 16 mt + 4 kg + r, r = 0..3 = the
        // window positions of pooled cell q = 4 mt + kg, for output channel co
#pragma unroll
        for (int i = 0; i < MPW; ++i) {
            const int q = 4 * (wm + 2 * i) + kg;
            if (q < HW && co < Co) {
                float best = acc[i][0] + bco;
                int sel = 0;
#pragma unroll
                for (int r = 1; r < 4; ++r) {
                    const float v = acc[i][r] + bco;
                    if (v > best) {
                        best = v;
                        sel = r;
                    }
                }
                const int o = (nb * Co + co) * HW + q;
                cur[o] = best;
                arg[o] = (uint8_t)sel;
            }
        }
        lds_barrier();  // done with col; the next image is staged
        nb += G;
        if (nb >= NB) break;
        buf ^= 1;
    }
}

// Weight gradient of a layer with few inputs per channel (Kc = Ci * 25 = KC
// <= 75: the network's input layer), straight from the pool's selection:
//   dW[co][k] = sum over pooled cells of dI times x under the selected output.
// Block (chunk, co) takes a fixed range of cells; each thread sums its cells
// in fp32, then a fixed-order tree over the block gives partial[chunk][co][k].
template <typename T, int KC>
__global__ __launch_bounds__(kThreads) void conv_dw_small_kernel(
    int Q, int cells, int Co, int H, int W, int Hp, int Wp, const float *__restrict__ dI,
    const uint8_t *__restrict__ arg, const T *__restrict__ x, float *__restrict__ partial) {
    constexpr int CI = KC / (KS * KS);
    __shared__ float red[KC][kThreads];
    const int co = blockIdx.y;
    const int q0 = blockIdx.x * cells, q1 = min(Q, q0 + cells);
    const int hw = Hp * Wp;
    float acc[KC];
#pragma unroll
    for (int k = 0; k < KC; ++k) acc[k] = 0.f;
    for (int q = q0 + threadIdx.x; q < q1; q += kThreads) {
        const int nb = q / hw, p = q - nb * hw, py = p / Wp, px = p - py * Wp;
        const int o = (nb * Co + co) * hw + p;
        const float g = dI[o];
        const int a = arg[o];
        const T *xp = x + (nb * CI * H + 2 * py + (a >> 1)) * W + 2 * px + (a & 1);
#pragma unroll
        for (int c = 0; c < CI; ++c)
#pragma unroll
            for (int ky = 0; ky < KS; ++ky)
#pragma unroll
                for (int kx = 0; kx < KS; ++kx) {
                    const int k = (c * KS + ky) * KS + kx;
                    acc[k] = __builtin_fmaf(g, (float)xp[(c * H + ky) * W + kx], acc[k]);
                }
    }
#pragma unroll
    for (int k = 0; k < KC; ++k) red[k][threadIdx.x] = acc[k];
    __syncthreads();
    for (int s = kThreads / 2; s > 0; s >>= 1) {
        if ((int)threadIdx.x < s) {
#pragma unroll
            for (int k = 0; k < KC; ++k) red[k][threadIdx.x] += red[k][threadIdx.x + s];
        }
        __syncthreads();
    }
    if ((int)threadIdx.x < KC)
        partial[(blockIdx.x * Co + co) * KC + threadIdx.x] = red[threadIdx.x][0];
}

// chunks of pooled cells per output channel for conv_dw_small_kernel: about
// 1024 workgroups in all (4 per compute unit); 4096 measured 12 % slower on
// the CSNN's first layer (more block reductions), 512 20 % slower
int small_dw_chunks(const ConvGeom &g, int64_t Q) {
    const int64_t by_cells = (Q + kThreads - 1) / kThreads;
    const int64_t by_grid = max(1, 1024 / g.Co);
    return (int)max((int64_t)1, min(by_cells, by_grid));
}

bool small_dw(const ConvGeom &g) { return g.Ci * KS * KS <= 75; }

// the input gradient by conv_dx_kernel (16-bit cores: not under fp32-only MFMA)
bool dx_one_pass(const ConvGeom &g, bool allow_split) {
    return allow_split && g.Ci * KS * KS <= kDxMaxK && g.Co <= kDxMaxCo &&
           g.Hp * g.Wp <= kDxMaxCells && g.H * g.W <= kDxThreads;
}

// the forward by conv_fwd_kernel and the weight gradient by conv_dw_kernel
// (spike input, exact in bf16; up to 32 pooled cells per channel)
bool dw_one_pass(const ConvGeom &g, int in_dtype, bool allow_split) {
    return in_dtype == SNN_U8 && allow_split && g.Ci * KS * KS <= kDxMaxK &&
           g.Co <= kDxMaxCo && g.Hp * g.Wp <= kFwMaxCells && g.H * g.W <= kDxThreads &&
           g.Ci * g.H * g.W % 4 == 0;  // images staged as 4-byte words
}

unsigned blocks(int64_t n) { return (unsigned)((n + kThreads - 1) / kThreads); }

// ---- plans and workspace ----------------------------------------------------
// forward:  [col (in dtype) Mw x ldk][C fp32 Mw x Co][gemm]
// backward: [dC^T fp32 Co x ldm] then, for dW, either [partial chunks x Co x Kc]
//           (few inputs per channel) or [planes 3 x Co x ldm][col^T Kc x ldm][gemm],
//           and, for dx (after dW), [dx^T fp32 Kc x ldm][gemm]

GemmArgs fwd_args(const ConvGeom &g, const ConvDims &v, int in_dtype, bool allow_split) {
    GemmArgs a{};
    a.M = (int)v.Mw; a.N = g.Co; a.K = v.Kc;
    a.lda = v.ldk; a.a_dtype = in_dtype; a.a_kc = true;
    a.ldb = v.Kc; a.b_dtype = SNN_F32; a.b_kc = true;
    a.ldc = g.Co; a.allow_split = allow_split;
    return a;
}

GemmArgs dw_args(const ConvGeom &g, const ConvDims &v, int in_dtype, bool allow_split) {
    GemmArgs a{};
    a.M = g.Co; a.N = v.Kc; a.K = (int)v.Mw;
    a.lda = v.ldm; a.a_dtype = kPlanes3; a.a_kc = true; a.a_ps = (int64_t)g.Co * v.ldm;
    a.ldb = v.ldm; a.b_dtype = in_dtype; a.b_kc = true;
    a.ldc = v.Kc; a.allow_split = allow_split;
    if (!(allow_split && gemm16_applies(a))) {
        a.a_dtype = SNN_F32;  // fp32 dC^T on the fp32 kernels
        a.a_ps = 0;
    }
    return a;
}

GemmArgs dx_args(const ConvGeom &g, const ConvDims &v, bool allow_split) {
    GemmArgs a{};
    a.M = v.Kc; a.N = (int)v.Mw; a.K = g.Co;
    a.lda = v.Kc; a.a_dtype = SNN_F32; a.a_kc = false;  // w[co][k]: k contiguous
    a.ldb = v.ldm; a.b_dtype = SNN_F32; a.b_kc = false;  // dC^T[co][m]: m contiguous
    a.ldc = v.ldm; a.allow_split = allow_split;
    return a;
}

size_t gemm_ws(const GemmArgs &a) {
    return gemm_workspace_bytes(a.M, a.N, a.K, a.a_dtype, a.b_dtype, a.a_kc, a.b_kc, a.allow_split);
}

struct BwdLayout {
    bool one_pass;  // weight gradient by conv_dw_kernel
    bool small;     // weight gradient by conv_dw_small_kernel
    int chunks;     // the partial sums of either
    size_t dct, partial, planes, colt, dw_gemm, dxt, dx_gemm;
    size_t dw_phase() const { return one_pass || small ? partial : planes + colt + dw_gemm; }
    size_t dx_phase() const { return dxt + dx_gemm; }
};

BwdLayout bwd_layout(const ConvGeom &g, const ConvDims &v, int in_dtype, bool allow_split) {
    BwdLayout l{};
    l.one_pass = dw_one_pass(g, in_dtype, allow_split);
    l.small = !l.one_pass && small_dw(g);
    l.dct = align_up((size_t)g.Co * v.ldm * sizeof(float));
    if (l.one_pass) {
        l.chunks = min(g.NB, kDwMaxGrid);
        l.partial = align_up((size_t)l.chunks * g.Co * v.Kc * sizeof(float));
    } else if (l.small) {
        l.chunks = small_dw_chunks(g, v.Q);
        l.partial = align_up((size_t)l.chunks * g.Co * v.Kc * sizeof(float));
    } else {
        const GemmArgs w = dw_args(g, v, in_dtype, allow_split);
        l.planes = w.a_dtype == kPlanes3 ? align_up((size_t)3 * g.Co * v.ldm * sizeof(uint16_t)) : 0;
        l.colt = align_up((size_t)v.Kc * v.ldm * dtype_bytes(in_dtype));
        l.dw_gemm = gemm_ws(w);
    }
    l.dxt = align_up((size_t)v.Kc * v.ldm * sizeof(float));
    l.dx_gemm = gemm_ws(dx_args(g, v, allow_split));
    return l;
}

template <typename T>
void launch_im2col(const ConvGeom &g, const ConvDims &v, const void *x, void *col, hipStream_t s) {
    if ((int64_t)g.Ci * g.H * g.W * (int64_t)sizeof(T) <= kIm2colLdsBytes && v.ldk <= kIm2colMaxK) {
        im2col_lds_kernel<T><<<(unsigned)g.NB, kThreads, 0, s>>>(
            v.Kc, (int)v.ldk, g.Ci, g.H, g.W, g.Hp, g.Wp, reinterpret_cast<const T *>(x),
            reinterpret_cast<T *>(col));
        return;
    }
    const int64_t n = v.Mw * (v.ldk / Chunk<T>::N);
    im2col_kernel<T><<<blocks(n), kThreads, 0, s>>>((int)v.Mw, v.Kc, (int)v.ldk, g.Ci, g.H, g.W,
                                                    g.Hp, g.Wp, reinterpret_cast<const T *>(x),
                                                    reinterpret_cast<T *>(col));
}

template <typename T>
void launch_im2col_t(const ConvGeom &g, const ConvDims &v, const void *x, void *colt,
                     hipStream_t s) {
    const int64_t n = (int64_t)v.Kc * (v.ldm / Chunk<T>::N);
    im2col_t_kernel<T><<<blocks(n), kThreads, 0, s>>>((int)v.Mw, v.Kc, (int)v.ldm, g.Ci, g.H, g.W,
                                                      g.Hp, g.Wp, reinterpret_cast<const T *>(x),
                                                      reinterpret_cast<T *>(colt));
}

template <typename T>
void launch_dw_small(const ConvGeom &g, const ConvDims &v, int chunks, const float *dI,
                     const uint8_t *arg, const void *x, float *partial, hipStream_t s) {
    const int cells = (int)((v.Q + chunks - 1) / chunks);
    dim3 grid((unsigned)chunks, (unsigned)g.Co);
    const T *xt = reinterpret_cast<const T *>(x);
    if (g.Ci == 1)
        conv_dw_small_kernel<T, 25><<<grid, kThreads, 0, s>>>((int)v.Q, cells, g.Co, g.H, g.W,
                                                              g.Hp, g.Wp, dI, arg, xt, partial);
    else if (g.Ci == 2)
        conv_dw_small_kernel<T, 50><<<grid, kThreads, 0, s>>>((int)v.Q, cells, g.Co, g.H, g.W,
                                                              g.Hp, g.Wp, dI, arg, xt, partial);
    else
        conv_dw_small_kernel<T, 75><<<grid, kThreads, 0, s>>>((int)v.Q, cells, g.Co, g.H, g.W,
                                                              g.Hp, g.Wp, dI, arg, xt, partial);
}

}  // namespace

bool conv_fits_int32(const ConvGeom &g) {
    const ConvDims v = dims_of(g);
    const int64_t lim = INT32_MAX;
    return (int64_t)g.NB * g.Ci * (g.H + 1) * (g.W + 1) <= lim && v.Mw * v.ldk <= lim &&
           (int64_t)v.Kc * v.ldm <= lim && (int64_t)g.Co * v.ldm <= lim && v.Mw * g.Co <= lim;
}

size_t conv_fwd_workspace_bytes(const ConvGeom &g, int in_dtype, bool allow_split) {
    const ConvDims v = dims_of(g);
    if (v.Mw == 0) return 0;
    return align_up((size_t)v.Mw * v.ldk * dtype_bytes(in_dtype)) +
           align_up((size_t)v.Mw * g.Co * sizeof(float)) +
           gemm_ws(fwd_args(g, v, in_dtype, allow_split));
}

size_t conv_bwd_workspace_bytes(const ConvGeom &g, int in_dtype, bool allow_split) {
    const ConvDims v = dims_of(g);
    if (v.Mw == 0) return 0;
    const BwdLayout l = bwd_layout(g, v, in_dtype, allow_split);
    return l.dct + max(l.dw_phase(), l.dx_phase());
}

hipError_t launch_conv_pool_fwd(const ConvGeom &g, const void *x, int in_dtype, const void *w,
                                const float *bias, float *cur, uint8_t *arg, bool allow_split,
                                void *ws, size_t ws_bytes, hipStream_t s) {
    const ConvDims v = dims_of(g);
    if (v.Mw == 0) return hipSuccess;
    if (ws == nullptr || ws_bytes < conv_fwd_workspace_bytes(g, in_dtype, allow_split))
        return hipErrorInvalidValue;
    if (!direct_conv(g) &&
        dw_one_pass(g, in_dtype, allow_split)) {
        const unsigned grid = (unsigned)min(g.NB, device_cus());
        const uint8_t *xb = reinterpret_cast<const uint8_t *>(x);
        const float *wf = reinterpret_cast<const float *>(w);
        if (g.Hp * g.Wp <= kDxMaxCells)
            conv_fwd_kernel<2><<<grid, kDxThreads, 0, s>>>(g.NB, g.Ci, g.H, g.W, g.Co, g.Hp, g.Wp,
                                                           xb, wf, bias, cur, arg);
        else
            conv_fwd_kernel<4><<<grid, kDxThreads, 0, s>>>(g.NB, g.Ci, g.H, g.W, g.Co, g.Hp, g.Wp,
                                                           xb, wf, bias, cur, arg);
        return hipGetLastError();
    }
    if (direct_conv(g)) {
        const float *wf = reinterpret_cast<const float *>(w);
        const uint8_t *xu = reinterpret_cast<const uint8_t *>(x);
        const float *xf = reinterpret_cast<const float *>(x);
        const unsigned grid = (unsigned)g.NB;
        if (in_dtype == SNN_U8 && g.Ci == 1)
            conv1_pool_kernel<uint8_t, 1><<<grid, kThreads, 0, s>>>(g.Ci, g.H, g.W, g.Co, g.Hp,
                                                                    g.Wp, xu, wf, bias, cur, arg);
        else if (in_dtype == SNN_U8)
            conv1_pool_kernel<uint8_t, kDirectMaxCi><<<grid, kThreads, 0, s>>>(
                g.Ci, g.H, g.W, g.Co, g.Hp, g.Wp, xu, wf, bias, cur, arg);
        else if (g.Ci == 1)
            conv1_pool_kernel<float, 1><<<grid, kThreads, 0, s>>>(g.Ci, g.H, g.W, g.Co, g.Hp, g.Wp,
                                                                  xf, wf, bias, cur, arg);
        else
            conv1_pool_kernel<float, kDirectMaxCi><<<grid, kThreads, 0, s>>>(
                g.Ci, g.H, g.W, g.Co, g.Hp, g.Wp, xf, wf, bias, cur, arg);
        return hipGetLastError();
    }
    char *p = reinterpret_cast<char *>(ws);
    void *col = p;
    p += align_up((size_t)v.Mw * v.ldk * dtype_bytes(in_dtype));
    float *C = reinterpret_cast<float *>(p);
    p += align_up((size_t)v.Mw * g.Co * sizeof(float));
    if (in_dtype == SNN_U8) launch_im2col<uint8_t>(g, v, x, col, s);
    else launch_im2col<float>(g, v, x, col, s);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    GemmArgs a = fwd_args(g, v, in_dtype, allow_split);
    a.A = col; a.B = w; a.C = C; a.bias = bias;
    // the contraction pools its own output when it can (else C, then the pool)
    bool pooled = false;
    a.pool_hw = g.Hp * g.Wp; a.pool_cur = cur; a.pool_arg = arg; a.pooled = &pooled;
    e = launch_gemm(a, p, ws_bytes - (size_t)(p - reinterpret_cast<char *>(ws)), s);
    if (e != hipSuccess) return e;
    if (pooled) return hipSuccess;
    const int S = g.Co | 1;
    const int QB = max(1, kPoolLdsFloats / (4 * S));
    pool_kernel<<<(unsigned)((v.Q + QB - 1) / QB), kThreads, 0, s>>>((int)v.Q, g.Co, g.Hp * g.Wp,
                                                                   QB, C, cur, arg);
    return hipGetLastError();
}

hipError_t launch_conv_pool_bwd(const ConvGeom &g, const float *dI, const uint8_t *arg,
                                const void *x, int in_dtype, const void *w, bool allow_split,
                                float *grad_w, float *grad_x, void *ws, size_t ws_bytes,
                                hipStream_t s) {
    const ConvDims v = dims_of(g);
    if (v.Mw == 0) return hipSuccess;
    if (ws == nullptr || ws_bytes < conv_bwd_workspace_bytes(g, in_dtype, allow_split))
        return hipErrorInvalidValue;
    const BwdLayout l = bwd_layout(g, v, in_dtype, allow_split);
    char *base = reinterpret_cast<char *>(ws);
    float *dct = reinterpret_cast<float *>(base);
    char *rest = base + l.dct;
    const size_t rest_bytes = ws_bytes - l.dct;
    hipError_t e;
    const bool dx1 = grad_x && dx_one_pass(g, allow_split);
    const bool dw_gemm = grad_w && !l.one_pass && !l.small;
    // dC^T in fp32 feeds the two-pass input gradient and an fp32 weight gradient
    const bool need_dct = (grad_x && !dx1) || (dw_gemm && l.planes == 0);
    if ((grad_x && !dx1) || dw_gemm) {
        uint16_t *planes = (dw_gemm && l.planes > 0) ? reinterpret_cast<uint16_t *>(rest) : nullptr;
        unpool_t_kernel<<<blocks(v.Q * g.Co), kThreads, 0, s>>>(
            (int)v.Q, g.Co, g.Hp * g.Wp, (int)v.ldm, dI, arg, need_dct ? dct : nullptr, planes);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (grad_w && l.one_pass) {
        float *partial = reinterpret_cast<float *>(rest);
        conv_dw_kernel<<<(unsigned)l.chunks, kDxThreads, 0, s>>>(
            g.NB, g.Ci, g.H, g.W, g.Co, g.Hp, g.Wp, dI, arg, reinterpret_cast<const uint8_t *>(x),
            partial);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        e = launch_splitk_reduce(g.Co, v.Kc, l.chunks, partial, grad_w, v.Kc, nullptr, s);
        if (e != hipSuccess) return e;
    } else if (grad_w && l.small) {
        float *partial = reinterpret_cast<float *>(rest);
        if (in_dtype == SNN_U8) launch_dw_small<uint8_t>(g, v, l.chunks, dI, arg, x, partial, s);
        else launch_dw_small<float>(g, v, l.chunks, dI, arg, x, partial, s);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        e = launch_splitk_reduce(g.Co, v.Kc, l.chunks, partial, grad_w, v.Kc, nullptr, s);
        if (e != hipSuccess) return e;
    } else if (grad_w) {
        char *colt = rest + l.planes;
        if (in_dtype == SNN_U8) launch_im2col_t<uint8_t>(g, v, x, colt, s);
        else launch_im2col_t<float>(g, v, x, colt, s);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        GemmArgs a = dw_args(g, v, in_dtype, allow_split);
        a.A = a.a_dtype == kPlanes3 ? static_cast<const void *>(rest) : dct;
        a.B = colt; a.C = grad_w; a.bias = nullptr;
        e = launch_gemm(a, colt + l.colt, rest_bytes - l.planes - l.colt, s);
        if (e != hipSuccess) return e;
    }
    if (dx1) {
        const unsigned grid = (unsigned)min(g.NB, device_cus());
        const int hw = g.H * g.W;  // at most 259 under dx_one_pass
        const float *wf = reinterpret_cast<const float *>(w);
        if (3 * hw <= kDxThreads)
            conv_dx_kernel<3><<<grid, kDxThreads, 0, s>>>(g.NB, g.Ci, g.H, g.W, g.Co, g.Hp, g.Wp,
                                                          dI, arg, wf, grad_x);
        else if (2 * hw <= kDxThreads)
            conv_dx_kernel<2><<<grid, kDxThreads, 0, s>>>(g.NB, g.Ci, g.H, g.W, g.Co, g.Hp, g.Wp,
                                                          dI, arg, wf, grad_x);
        else
            conv_dx_kernel<1><<<grid, kDxThreads, 0, s>>>(g.NB, g.Ci, g.H, g.W, g.Co, g.Hp, g.Wp,
                                                          dI, arg, wf, grad_x);
        return hipGetLastError();
    }
    if (grad_x) {
        float *dxt = reinterpret_cast<float *>(rest);
        GemmArgs a = dx_args(g, v, allow_split);
        a.A = w; a.B = dct; a.C = dxt; a.bias = nullptr;
        e = launch_gemm(a, rest + l.dxt, rest_bytes - l.dxt, s);
        if (e != hipSuccess) return e;
        const int PH = (g.H + 1) / 2, PW = (g.W + 1) / 2;
        const int total = g.NB * g.Ci * PH * PW * 4;
        col2im_kernel<<<blocks(total), kThreads, 0, s>>>(total, g.Ci, g.H, g.W, PH, PW, g.Hp, g.Wp,
                                                         (int)v.ldm, dxt, grad_x);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace snn
