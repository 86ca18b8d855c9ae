// The whole training step of a two-layer dense SNN in one launch, for small
// batches, where a step of separate kernels is a chain of launch latencies
// (Sec. IV's small-batch results): a hidden layer n_in -> n_hid (Leaky or
// Synaptic, spike input) and a readout n_hid -> n_out whose spike counts feed
// the loss (Sec. V), forward, loss and BPTT backward (eqs. 3-9).
//
// Neuron-parallel: workgroup w owns NPW consecutive hidden neurons and runs
// everything that touches only them: their currents, forward scan, reverse
// scan, and their rows of dW0 and db0 and columns of dW1, with the currents,
// membrane, spikes and dL/dI of its neurons in LDS the whole time.  Three
// grid barriers separate the phases:
//   0  (all)  the input spikes packed to bits, a slice per workgroup (every
//             workgroup reads all of x twice, 8 times fewer bytes so);
//                                                          -- barrier 1 --
//   A  (all)  I0 = x W0^T + b0 for the own neurons, forward scan; spikes to
//             global memory;                               -- barrier 2 --
//   B  (one workgroup per sample) readout currents, readout forward scan,
//             loss and dL/dcounts, readout reverse scan -> dI1;  -- barrier 3 --
//   C  (all)  the readout's input gradient folded into the hidden reverse scan
//             (g0 = dI1 W1 per step), dW0, db0, dW1 of the own neurons;
//             workgroup 0 also db1 and the batch loss.
// Every operand a phase reads from global memory is first staged in LDS with
// all its loads in flight at once.  The three contractions (hidden currents,
// readout currents, dW0) run on v_mfma_f32_16x16x32_bf16 with the exact
// products of the layer calls: spikes are exact in bf16, fp32 values are
// split into three exact bf16 parts (hi, mid, lo; the smallest multiplied
// first), accumulation in fp32.  The scans and adjoints use the time scans'
// arithmetic (neuron.hpp); db, dW1 and the fold accumulate in fp32.
//
// Fragments (16x16x32): lane l supplies 8 values of row l % 16 of A and of
// column l % 16 of B at k = 8 (l / 16) + e of the step; it receives rows
// 4 (l / 16) + i of column l % 16 of the result.
//
// Grid barriers count arrivals on a device counter (agent-scope atomics).
// What one workgroup hands to another is stored write-through (agent-scope
// atomic stores) and read after an agent-scope acquire fence, so it is seen
// across XCDs without writing back any L2.  The grid is at most one
// workgroup per compute unit, so all of it is resident at once on an
// otherwise idle device; every wait is bounded all the same: after
// wait_limit polls the workgroup marks the step failed in *status and skips
// the rest of the step, so the launch ends instead of hanging.  Every
// workgroup counts its exit on a second counter and the last one clears
// both, so the counters are zero again after every launch, also a failed
// one.  Calls that overlap on one device share the counters and must not be
// made.
#include <atomic>

#include "neuron.hpp"

namespace snn {

namespace {

constexpr int kThreads = 512;  // 8 waves
constexpr int kWaves = kThreads / 64;
constexpr unsigned kDefaultWaitLimit = 1u << 22;  // polls of ~100 cycles: well over 0.1 s

// arrivals, exits
__device__ unsigned g_fused_bar[2];

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

struct FusedArgs {
    int T, B, n_in, n_hid, n_out, K, P;
    int neuron0, neuron1;
    bool rs0, rs1;  // reset differentiated through the surrogate
    float alpha0, beta0, thr0, slope0, alpha1, beta1, thr1, slope1;
    int loss_kind;
    unsigned wait_limit;
    const uint8_t *x;
    const float *W0, *b0, *W1, *b1;
    const int32_t *labels;
    const float *targets;
    float *loss, *counts, *gW0, *gb0, *gW1, *gb1;
    uint8_t *spk;  // [T][B][n_hid] hidden spikes out, or NULL
    int32_t *status;
    uint8_t *xb;    // [R][n_in / 8] input spikes as bits (bit e of byte k: input 8 k + e)
    uint8_t *s0;    // [B][T][hid_stride] hidden spikes handed to the readout
    float *dI1;     // [R][n_out] readout dL/dI
    double *lossb;  // [B] per-sample loss terms
};

__host__ __device__ inline size_t up16(size_t n) { return (n + 15) & ~(size_t)15; }
__host__ __device__ inline int round32(int n) { return (n + 31) & ~31; }
// hidden spike rows in global memory and LDS: [T][hid_stride(n_hid)] bytes per
// sample, whole 32-wide k-steps (the padding columns meet zero weights)
__host__ __device__ inline int hid_stride(int n_hid) { return round32(n_hid); }

// LDS carve-up (bytes), the same on host and device.  Region X: the packed
// input (phases A and C) or phase B's sample (spike rows [T][hid_stride], W1
// [n_out][hid_stride], readout currents, membrane, class values and partial
// sums).  Region Y: the bf16 parts of the own neurons' W0 rows [3][NPW][kp]
// (phase A) or the staged dI1 [R][n_out] (phase C).  Then W1 columns of the own neurons and
// the own neurons' state.
struct FusedLds {
    size_t y, bw, bi, bu, bc;  // region Y; phase B offsets in region X
    size_t wc, il, ul, sl, total;
};

__host__ __device__ inline size_t xbits_bytes(int T, int B, int n_in) {
    return up16((size_t)T * B * (n_in / 8));
}

__host__ __device__ inline FusedLds fused_lds(int T, int B, int n_in, int n_hid, int n_out,
                                              int npw) {
    const size_t R = (size_t)T * B;
    FusedLds l{};
    l.bw = up16((size_t)T * hid_stride(n_hid));
    l.bi = l.bw + up16((size_t)n_out * hid_stride(n_hid) * 4);
    l.bu = l.bi + up16((size_t)T * n_out * 4);
    l.bc = l.bu + up16((size_t)T * n_out * 4);
    const size_t xb = xbits_bytes(T, B, n_in), phb = l.bc + 64 * 8 + 4 * 32 * 16 * 4;
    l.y = up16(xb > phb ? xb : phb);
    const size_t wf = 3 * (size_t)npw * round32(n_in) * 2, d1 = R * n_out * 4;
    l.wc = l.y + up16(wf > d1 ? wf : d1);
    l.il = l.wc + up16((size_t)npw * kFusedMaxOut * 4);  // [NPW][16] W1 columns
    l.ul = l.il + up16(R * npw * 4);  // [R][NPW] fp32 membrane (il: currents, then dI0)
    l.sl = l.ul + up16(R * npw * 4);  // [R][NPW] u8 spikes
    l.total = l.sl + up16(R * npw);
    return l;
}

// Copy n 16-byte chunks from global memory to LDS with every thread, 8
// chunks in flight per thread (clamped, so that every load is issued at once).
// Workgroups that copy the same array start at different chunks (workgroup w
// of G at chunk w n / G, wrapping around), so that their requests spread over
// the memory channels instead of all hitting the same lines at once.
__device__ inline void stage16(void *dst, const void *src, int n) {
    const u32x4 *s = reinterpret_cast<const u32x4 *>(src);
    u32x4 *d = reinterpret_cast<u32x4 *>(dst);
    const int rot = (int)(((int64_t)blockIdx.x * n) / gridDim.x);
    auto at = [&](int i) { const int j = i + rot; return j >= n ? j - n : j; };
    for (int base = threadIdx.x; base < n; base += kThreads * 8) {
        u32x4 v[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) v[k] = s[at(min(base + k * kThreads, n - 1))];
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            const int i = base + k * kThreads;
            if (i < n) d[at(i)] = v[k];
        }
    }
}

__device__ inline double wave_sum(double v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}
__device__ inline double wave_max(double v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v = fmax(v, __shfl_xor(v, off, 64));
    return v;
}

// ---- MFMA operands -----------------------------------------------------------
__device__ inline uint32_t bf16_bits(float x) {  // round to nearest even (finite x)
    const uint32_t b = __float_as_uint(x);
    return (b + 0x7fffu + ((b >> 16) & 1u)) >> 16;
}

// 8 fp32 values as three exact bf16 parts (p[0] = hi, p[1] = mid, p[2] = lo)
__device__ inline void split3(const float (&v)[8], u32x4 (&p)[3]) {
    uint32_t h[3][8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        h[0][e] = bf16_bits(v[e]);
        const float r = v[e] - __uint_as_float(h[0][e] << 16);
        h[1][e] = bf16_bits(r);
        h[2][e] = bf16_bits(r - __uint_as_float(h[1][e] << 16));
    }
#pragma unroll
    for (int k = 0; k < 3; ++k)
        p[k] = u32x4{h[k][0] | (h[k][1] << 16), h[k][2] | (h[k][3] << 16),
                     h[k][4] | (h[k][5] << 16), h[k][6] | (h[k][7] << 16)};
}

// 8 bytes (little-endian in w0, w1) as bf16 (every byte value is exact)
__device__ inline u32x4 bytes_bf16(uint32_t w0, uint32_t w1) {
    uint32_t o[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint32_t w = i < 2 ? w0 : w1;
        const float lo = (float)((w >> (16 * (i % 2))) & 0xffu);
        const float hi = (float)((w >> (16 * (i % 2) + 8)) & 0xffu);
        o[i] = (__float_as_uint(lo) >> 16) | (__float_as_uint(hi) & 0xffff0000u);
    }
    return u32x4{o[0], o[1], o[2], o[3]};
}

// 8 bits (bit e: value e) as bf16 0 / 1
__device__ inline u32x4 bits_bf16(uint32_t bits) {
    uint32_t o[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
        o[i] = ((bits >> (2 * i)) & 1u ? 0x3f80u : 0u) |
               ((bits >> (2 * i + 1)) & 1u ? 0x3f800000u : 0u);
    return u32x4{o[0], o[1], o[2], o[3]};
}

// bit Q of 8 bytes (byte e: value e) as bf16 0 / 1
template <int Q>
__device__ inline u32x4 bitcol_bf16(const uint32_t (&b)[8]) {
    uint32_t o[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
        o[i] = ((b[2 * i] >> Q) & 1u ? 0x3f80u : 0u) | ((b[2 * i + 1] >> Q) & 1u ? 0x3f800000u : 0u);
    return u32x4{o[0], o[1], o[2], o[3]};
}

__device__ inline floatx4 mfma(const u32x4 &a, const u32x4 &b, const floatx4 &c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// A (one 16-bit part) against the three parts of B, smallest first
__device__ inline floatx4 mfma3(const u32x4 &a, const u32x4 (&b)[3], floatx4 c) {
    c = mfma(a, b[2], c);
    c = mfma(a, b[1], c);
    return mfma(a, b[0], c);
}

// ---- grid barrier ---------------------------------------------------------------
// Values one workgroup hands to others (hidden spikes, readout dL/dI, loss
// terms) are stored with agent-scope atomic stores, which write through the
// XCD's L2, so a barrier needs no L2 writeback: each wave waits for its own
// stores, then thread 0 counts the workgroup in.
template <typename V>
__device__ inline void put_shared(V *p, V v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Grid barrier number k (1, 2): returns false if the wait gave up.  After it
// an agent-scope acquire fence drops this CU's and XCD's cached copies, so
// the other workgroups' shared values are read from memory.
__device__ inline bool grid_barrier(unsigned k, unsigned G, unsigned limit, int32_t *status,
                                    bool *ok) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (threadIdx.x == 0) {
        __hip_atomic_fetch_add(&g_fused_bar[0], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        unsigned n = 0;
        bool good = true;
        while (__hip_atomic_load(&g_fused_bar[0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) <
               k * G) {
            if (++n > limit) {
                good = false;
                __hip_atomic_store(status, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                break;
            }
            __builtin_amdgcn_s_sleep(1);
        }
        *ok = good;
    }
    __syncthreads();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    return *ok;
}

// one forward step / one adjoint step of layer 0 (hidden) or 1 (readout)
__device__ inline float step_fwd(const FusedArgs &a, int layer, float &u, float &syn, float zp,
                                 float in) {
    const bool syn_n = (layer == 0 ? a.neuron0 : a.neuron1) == SNN_SYNAPTIC;
    const float al = layer == 0 ? a.alpha0 : a.alpha1, be = layer == 0 ? a.beta0 : a.beta1,
                jump = layer == 0 ? -a.thr0 : -a.thr1;
    return syn_n ? neuron_step<SNN_SYNAPTIC>(u, syn, zp, in, al, be, jump)
                 : neuron_step<SNN_LEAKY>(u, syn, zp, in, al, be, jump);
}

__device__ inline float step_adj(const FusedArgs &a, int layer, float &lam, float &lami, float g,
                                 float s) {
    const bool syn = (layer == 0 ? a.neuron0 : a.neuron1) == SNN_SYNAPTIC;
    const bool rs = layer == 0 ? a.rs0 : a.rs1;
    const float al = layer == 0 ? a.alpha0 : a.alpha1, be = layer == 0 ? a.beta0 : a.beta1,
                th = layer == 0 ? a.thr0 : a.thr1;
    if (syn)
        return rs ? adjoint_step<SNN_SYNAPTIC, true>(lam, lami, g, s, al, be, th)
                  : adjoint_step<SNN_SYNAPTIC, false>(lam, lami, g, s, al, be, th);
    return rs ? adjoint_step<SNN_LEAKY, true>(lam, lami, g, s, al, be, th)
              : adjoint_step<SNN_LEAKY, false>(lam, lami, g, s, al, be, th);
}

template <int NPW>
__global__ __launch_bounds__(kThreads) void fused_step_kernel(FusedArgs a) {
    static_assert(NPW <= 16, "the own neurons are one 16-wide MFMA block");
    extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
    __shared__ bool ok;
    __shared__ float red[kThreads];
    const int G = gridDim.x, w = blockIdx.x, tid = threadIdx.x;
    const int lane = tid & 63, wv = tid >> 6, col = lane & 15, kg = lane >> 4;
    const int T = a.T, B = a.B, n_in = a.n_in, n_hid = a.n_hid, n_out = a.n_out;
    const int R = T * B, NB = n_in / 8;  // packed bytes per input row
    const int o0 = w * NPW, nq = min(NPW, n_hid - o0);
    const FusedLds L = fused_lds(T, B, n_in, n_hid, n_out, NPW);
    const int HS = hid_stride(n_hid);
    uint8_t *Xb = lds;                                          // region X: [R][NB] bits
    float *Wc = reinterpret_cast<float *>(lds + L.wc);          // [NPW][16]
    float *Il = reinterpret_cast<float *>(lds + L.il);
    float *Ul = reinterpret_cast<float *>(lds + L.ul);
    uint8_t *Sl = lds + L.sl;
    const unsigned limit = a.wait_limit;
    const int nxb = (int)(xbits_bytes(T, B, n_in) / 16);  // 16-byte chunks of packed x
    if (w == 0 && tid == 0) __hip_atomic_store(a.status, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    // W1 rows [n_out][HS] for the readout phase (workgroups w < B)
    float *W1l = reinterpret_cast<float *>(lds + L.bw);
    auto stage_w1 = [&] {
        if (w >= B) return;
        // W1 rows at stride HS: 16-byte chunks when rows are whole chunks
        if (n_hid % 4 == 0) {
            const int cpr = n_hid / 4, nc = n_out * cpr;
            const u32x4 *src = reinterpret_cast<const u32x4 *>(a.W1);
            for (int i0 = tid; i0 < nc; i0 += 8 * kThreads) {
                u32x4 v[8];
#pragma unroll
                for (int k = 0; k < 8; ++k) v[k] = src[min(i0 + k * kThreads, nc - 1)];
#pragma unroll
                for (int k = 0; k < 8; ++k) {
                    const int i = i0 + k * kThreads;
                    if (i < nc)
                        *reinterpret_cast<u32x4 *>(W1l + (i / cpr) * HS + 4 * (i % cpr)) = v[k];
                }
            }
        } else {
            for (int i = tid; i < n_out * n_hid; i += kThreads)
                W1l[(i / n_hid) * HS + i % n_hid] = a.W1[i];
        }
    };
    // W1 rows go in with the W0 parts when they do not overlap the packed
    // input of phase A (region X: packed input, then phase B's sample)
    const bool w1_early = xbits_bytes(T, B, n_in) <= L.bw;

    // ---- 0: the input spikes as bits, 4 packed bytes (32 inputs) per thread
    {
        const int64_t nf = (int64_t)R * NB;  // packed bytes; x byte 8 f + e is bit e of f
        const int64_t n4 = (nf + 3) / 4, per = (n4 + G - 1) / G;
        for (int64_t i = (int64_t)w * per + tid; i < min(n4, (int64_t)(w + 1) * per); i += kThreads) {
            uint32_t word = 0;
#pragma unroll
            for (int h = 0; h < 4; ++h) {
                const int64_t f = 4 * i + h;
                if (f < nf) {
                    const uint2 v = *reinterpret_cast<const uint2 *>(a.x + 8 * f);
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const uint32_t byte = ((e < 4 ? v.x : v.y) >> (8 * (e % 4))) & 0xffu;
                        word |= (byte != 0u ? 1u : 0u) << (8 * h + e);
                    }
                }
            }
            put_shared(reinterpret_cast<uint32_t *>(a.xb) + i, word);
        }
    }
    const int kp = round32(n_in);
    uint16_t *Wp = reinterpret_cast<uint16_t *>(lds + L.y);  // [3][NPW][kp]
    {
        // the bf16 parts of the own neurons' W0 rows (zero past n_in and past
        // the last neuron) and W1 columns of the own neurons: LDS is free and
        // W0 does not depend on phase 0, so their loads run before barrier 1
        for (int i0 = tid; i0 < kp; i0 += 4 * kThreads) {
            float v[NPW][4];
#pragma unroll
            for (int q = 0; q < NPW; ++q)
#pragma unroll
                for (int k = 0; k < 4; ++k)
                    v[q][k] = a.W0[(int64_t)(o0 + min(q, nq - 1)) * n_in +
                                   min(i0 + k * kThreads, n_in - 1)];
#pragma unroll
            for (int q = 0; q < NPW; ++q)
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const int i = i0 + k * kThreads;
                    if (i < kp) {
                        const float x = (q < nq && i < n_in) ? v[q][k] : 0.f;
                        const uint32_t hi = bf16_bits(x);
                        const float r = x - __uint_as_float(hi << 16);
                        const uint32_t mid = bf16_bits(r);
                        Wp[(0 * NPW + q) * kp + i] = (uint16_t)hi;
                        Wp[(1 * NPW + q) * kp + i] = (uint16_t)mid;
                        Wp[(2 * NPW + q) * kp + i] = (uint16_t)bf16_bits(r - __uint_as_float(mid << 16));
                    }
                }
        }
        if (tid < NPW * kFusedMaxOut) {
            const int q = tid / kFusedMaxOut, j = tid % kFusedMaxOut;
            Wc[tid] = (q < nq && j < n_out) ? a.W1[(int64_t)j * n_hid + o0 + q] : 0.f;
        }
        if (w1_early) stage_w1();
    }
    bool alive = grid_barrier(1, G, limit, a.status, &ok);

    // ---- A: currents and forward scan of the own neurons ---------------------
    if (alive) {
        stage16(Xb, a.xb, nxb);
        __syncthreads();
        // D[r][q] = sum_k x[r][k] W0[o0 + q][k]: wave wv takes row blocks wv,
        // wv + kWaves, ..., kGroup of them at a time; per k-step the blocks'
        // MFMAs of one part follow each other (independent accumulators)
        constexpr int kGroup = 4;
        const int KS = kp / 32, RB = (R + 15) / 16;
        for (int g = 0; kWaves * kGroup * g + wv < RB; ++g) {
            auto blk = [&](int j) { return kWaves * (kGroup * g + j) + wv; };
            floatx4 acc[kGroup];
#pragma unroll
            for (int j = 0; j < kGroup; ++j) acc[j] = floatx4{0.f, 0.f, 0.f, 0.f};
            for (int ks = 0; ks < KS; ++ks) {
                const int kb = ks * 4 + kg;  // packed byte: inputs 8 kb .. 8 kb + 7
                u32x4 bp[3];
#pragma unroll
                for (int p = 0; p < 3; ++p)
                    bp[p] = col < NPW ? *reinterpret_cast<const u32x4 *>(Wp + (p * NPW + col) * kp + 8 * kb)
                                      : u32x4{0u, 0u, 0u, 0u};
                u32x4 av[kGroup];
#pragma unroll
                for (int j = 0; j < kGroup; ++j) {
                    const int r = blk(j) * 16 + col;
                    av[j] = bits_bf16((r < R && kb < NB) ? Xb[r * NB + kb] : 0u);
                }
#pragma unroll
                for (int p = 2; p >= 0; --p)
#pragma unroll
                    for (int j = 0; j < kGroup; ++j)
                        if (blk(j) < RB) acc[j] = mfma(av[j], bp[p], acc[j]);
            }
            const float bq = (col < nq && a.b0) ? a.b0[o0 + col] : 0.f;
#pragma unroll
            for (int j = 0; j < kGroup; ++j)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int r = blk(j) * 16 + 4 * kg + i;
                    if (r < R && col < NPW) Il[r * NPW + col] = acc[j][i] + bq;
                }
        }
        __syncthreads();
        // one thread per own column (b, q), neurons fastest: consecutive
        // threads read consecutive LDS words and store consecutive spikes
        for (int c = tid; c < nq * B; c += kThreads) {
            const int b = c / nq, q = c % nq, o = o0 + q;
            float u = 0.f, syn = 0.f, zp = 0.f;
            for (int t = 0; t < T; ++t) {
                const int r = t * B + b;
                const float uu = step_fwd(a, 0, u, syn, zp, Il[r * NPW + q]);
                zp = uu > a.thr0 ? 1.f : 0.f;
                Ul[r * NPW + q] = uu;
                Sl[r * NPW + q] = (uint8_t)zp;
                put_shared(&a.s0[((int64_t)b * T + t) * HS + o], (uint8_t)zp);
                if (a.spk) a.spk[(int64_t)r * n_hid + o] = (uint8_t)zp;
            }
        }
        alive = grid_barrier(2, G, limit, a.status, &ok);
    }

    // ---- B: readout forward, loss, readout reverse scan (one sample each) ----
    if (alive) {
        uint8_t *Sb = lds;                                       // [T][HS]
        float *I1 = reinterpret_cast<float *>(lds + L.bi);       // [T][n_out]
        float *U1 = reinterpret_cast<float *>(lds + L.bu);       // [T][n_out]
        double *cls = reinterpret_cast<double *>(lds + L.bc);    // [64]
        float *part = reinterpret_cast<float *>(cls + 64);       // [4][32][16] k-quarter partials
        if (!w1_early) stage_w1();
        for (int b = w; b < B; b += G) {
            __syncthreads();
            stage16(Sb, a.s0 + (int64_t)b * T * HS, T * HS / 16);
            __syncthreads();
            // D[t][j] = sum_o s[t][o] W1[j][o]: wave wv takes row block wv & 1
            // (t < 32) and quarter wv >> 1 of the k-steps; the quarters are
            // added in order
            {
                const int tb = wv & 1, half = wv >> 1;
                const int KS = HS / 32, kh = (KS + 3) / 4;
                const int ks0 = half * kh, ks1 = min(KS, ks0 + kh);
                const int t = tb * 16 + col;
                floatx4 acc = floatx4{0.f, 0.f, 0.f, 0.f};
                for (int ks = ks0; ks < ks1; ++ks) {
                    const int k = ks * 32 + 8 * kg;
                    const uint2 sv = t < T ? *reinterpret_cast<const uint2 *>(Sb + t * HS + k)
                                           : make_uint2(0u, 0u);
                    float wv8[8];
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        wv8[e] = (col < n_out && k < n_hid) ? W1l[col * HS + k + e] : 0.f;
                    u32x4 bp[3];
                    split3(wv8, bp);
                    acc = mfma3(bytes_bf16(sv.x, sv.y), bp, acc);  // one chain: T <= 32
                }
#pragma unroll
                for (int i = 0; i < 4; ++i) part[(half * 32 + tb * 16 + 4 * kg + i) * 16 + col] = acc[i];
            }
            __syncthreads();
            for (int idx = tid; idx < T * n_out; idx += kThreads) {
                const int t = idx / n_out, j = idx % n_out;
                I1[idx] = (((part[t * 16 + j] + part[(32 + t) * 16 + j]) + part[(64 + t) * 16 + j]) +
                           part[(96 + t) * 16 + j]) + (a.b1 ? a.b1[j] : 0.f);
            }
            __syncthreads();
            if (tid < 64) {
                const int j = tid;
                const bool has = j < n_out;
                float u = 0.f, syn = 0.f, zp = 0.f, cnt = 0.f;
                if (has) {
                    for (int t = 0; t < T; ++t) {
                        const float uu = step_fwd(a, 1, u, syn, zp, I1[t * n_out + j]);
                        zp = uu > a.thr1 ? 1.f : 0.f;
                        cnt += zp;
                        U1[t * n_out + j] = uu;
                    }
                    if (a.counts) a.counts[(int64_t)b * n_out + j] = cnt;
                }
                red[j] = cnt;
                __builtin_amdgcn_wave_barrier();
                // class k = lane: the count of its population (exact in fp64)
                const int K = a.K, P = a.P, k = j;
                const bool cl = k < K;
                double c = 0.0;
                if (cl)
                    for (int p = 0; p < P; ++p) c += (double)red[k * P + p];
                double lb, gk;
                if (a.loss_kind == SNN_LOSS_CE_COUNT) {
                    const int y = a.labels[b];
                    const bool good = y >= 0 && y < K;
                    const double mx = wave_max(cl ? c : -__builtin_inf());
                    const double e = cl ? exp(c - mx) : 0.0;
                    const double se = wave_sum(e);
                    const double cy = __shfl(c, good ? y : 0, 64);
                    lb = good ? (mx + log(se)) - cy : __builtin_nan("");
                    gk = good ? (e / se - (k == y ? 1.0 : 0.0)) / (double)a.B : __builtin_nan("");
                } else {
                    const double d = cl ? c - (double)a.targets[(int64_t)b * K + k] : 0.0;
                    lb = wave_sum(d * d);
                    gk = 2.0 * d / ((double)a.B * K);
                }
                if (j == 0) put_shared(&a.lossb[b], lb);
                cls[j] = gk;
                __builtin_amdgcn_wave_barrier();
                if (has) {
                    const float g = (float)cls[j / P];
                    float lam = 0.f, lami = 0.f;
                    for (int t = T - 1; t >= 0; --t) {
                        const float s = surrogate(U1[t * n_out + j], a.thr1, a.slope1);
                        put_shared(&a.dI1[(int64_t)(t * B + b) * n_out + j],
                                   step_adj(a, 1, lam, lami, g, s));
                    }
                }
            }
        }
        alive = grid_barrier(3, G, limit, a.status, &ok);
    }

    // ---- C: hidden reverse scan with the folded readout gradient, gradients --
    if (alive) {
        float *D1 = reinterpret_cast<float *>(lds + L.y);  // [R][n_out]
        stage16(D1, a.dI1, R * n_out / 4);
        for (int i = (R * n_out / 4) * 4 + tid; i < R * n_out; i += kThreads) D1[i] = a.dI1[i];
        stage16(Xb, a.xb, nxb);
        __syncthreads();
        for (int c = tid; c < nq * B; c += kThreads) {
            const int b = c / nq, q = c % nq;
            float wcol[kFusedMaxOut];
#pragma unroll
            for (int j = 0; j < kFusedMaxOut; ++j) wcol[j] = Wc[q * kFusedMaxOut + j];
            float lam = 0.f, lami = 0.f;
            for (int t = T - 1; t >= 0; --t) {
                const int r = t * B + b;
                // dL/dz_t = sum_j dI1[t,b,j] W1[j,o], j ascending (the weights
                // past n_out are 0: their reads are clamped into the array)
                float dv[kFusedMaxOut];
#pragma unroll
                for (int j = 0; j < kFusedMaxOut; ++j) dv[j] = D1[min(r * n_out + j, R * n_out - 1)];
                float gt = 0.f;
#pragma unroll
                for (int j = 0; j < kFusedMaxOut; ++j) gt = __builtin_fmaf(dv[j], wcol[j], gt);
                const float s = surrogate(Ul[r * NPW + q], a.thr0, a.slope0);
                Il[r * NPW + q] = step_adj(a, 0, lam, lami, gt, s);  // the currents are spent
            }
        }
        __syncthreads();
        // db0: rows ascending
        if (tid < nq && a.gb0) {
            float s = 0.f;
            for (int r = 0; r < R; ++r) s += Il[r * NPW + tid];
            a.gb0[o0 + tid] = s;
        }
        // dW0[o0 + q][n] = sum_r dI0[r][q] x[r][n]: A = dI0 (the own neurons as
        // rows, three parts), B = x; a lane reads the packed byte of columns
        // n .. n + 7 (n = n_w + 8 col) of each of its 8 rows and forms the
        // operands of columns n + Q, Q = 0..7: three MFMAs per Q, 128 columns
        // per group; wave wv takes groups wv, wv + kWaves, ...
        if (a.gW0) {
            const int NG = (n_in + 127) / 128, KR = (R + 31) / 32;
            for (int gi = wv; gi < NG; gi += kWaves) {
                const int nb = gi * 16 + col;  // packed byte of the lane's 8 columns
                floatx4 acc[8];
#pragma unroll
                for (int q = 0; q < 8; ++q) acc[q] = floatx4{0.f, 0.f, 0.f, 0.f};
                for (int ks = 0; ks < KR; ++ks) {
                    uint32_t xr[8];
                    float dv[8];
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const int r = ks * 32 + 8 * kg + e;
                        xr[e] = (r < R && nb < NB) ? Xb[r * NB + nb] : 0u;
                        dv[e] = (col < nq && r < R) ? Il[r * NPW + min(col, NPW - 1)] : 0.f;
                    }
                    u32x4 ap[3];
                    split3(dv, ap);
                    u32x4 bq[8];
                    bq[0] = bitcol_bf16<0>(xr); bq[1] = bitcol_bf16<1>(xr);
                    bq[2] = bitcol_bf16<2>(xr); bq[3] = bitcol_bf16<3>(xr);
                    bq[4] = bitcol_bf16<4>(xr); bq[5] = bitcol_bf16<5>(xr);
                    bq[6] = bitcol_bf16<6>(xr); bq[7] = bitcol_bf16<7>(xr);
#pragma unroll
                    for (int p = 2; p >= 0; --p)
#pragma unroll
                        for (int Q = 0; Q < 8; ++Q) acc[Q] = mfma(ap[p], bq[Q], acc[Q]);
                }
                // result rows 4 kg + i are the neurons, column col the byte
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int q = 4 * kg + i;
                    if (q < nq && nb < NB)
#pragma unroll
                        for (int Q = 0; Q < 8; ++Q) a.gW0[(int64_t)(o0 + q) * n_in + 8 * nb + Q] = acc[Q][i];
                }
            }
        }
        // dW1 columns of the own neurons: output (j, q) split over row groups
        if (a.gW1) {
            const int nout = n_out * nq;  // at most 16 * 16
            const int groups = max(1, kThreads / nout), per = (R + groups - 1) / groups;
            float part = 0.f;
            if (tid < nout * groups) {
                const int id = tid % nout, gi = tid / nout, j = id / nq, q = id % nq;
                for (int r = gi * per; r < min(R, (gi + 1) * per); ++r)
                    part = __builtin_fmaf(D1[r * n_out + j], (float)Sl[r * NPW + q], part);
            }
            red[tid] = part;
            __syncthreads();
            if (tid < nout) {
                float s = 0.f;
                for (int g = 0; g < groups; ++g) s += red[g * nout + tid];
                a.gW1[(int64_t)(tid / nq) * n_hid + o0 + tid % nq] = s;
            }
        }
        if (w == 0) {
            if (a.gb1 && tid < n_out) {
                float s = 0.f;
                for (int r = 0; r < R; ++r) s += D1[r * n_out + tid];
                a.gb1[tid] = s;
            }
            if (tid == 0 && a.loss) {
                double s = 0.0;
                for (int b = 0; b < B; ++b) s += a.lossb[b];
                *a.loss = (float)(a.loss_kind == SNN_LOSS_CE_COUNT ? s / (double)B
                                                                    : s / ((double)B * a.K));
            }
        }
    }

    // exit: the last workgroup out clears the counters for the next launch
    __syncthreads();
    if (tid == 0) {
        // no data is published through the counters: relaxed order suffices
        const unsigned prev =
            __hip_atomic_fetch_add(&g_fused_bar[1], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (prev == (unsigned)G - 1) {
            __hip_atomic_store(&g_fused_bar[0], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(&g_fused_bar[1], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
}

template <int NPW>
void *kernel_of() { return reinterpret_cast<void *>(&fused_step_kernel<NPW>); }

}  // namespace

FusedPlan fused_plan(int T, int B, int n_in, int n_hid, int n_out) {
    FusedPlan p{};
    const int cus = device_cus();
    // the most neurons per workgroup (up to 16: the contractions cost the
    // same for any of these) whose state fits in LDS, with a grid that fits
    // the device
    for (int npw = kFusedMaxNpw; npw >= 4; npw /= 2) {
        const size_t lds = fused_lds(T, B, n_in, n_hid, n_out, npw).total;
        if (lds <= kFusedMaxLds && (n_hid + npw - 1) / npw <= cus) {
            p.ok = true;
            p.npw = npw;
            p.lds = lds;
            break;
        }
    }
    p.grid = p.ok ? (n_hid + p.npw - 1) / p.npw : 0;
    const size_t R = (size_t)T * B;
    p.ws_bytes = align_up(R * hid_stride(n_hid)) + align_up(R * n_out * sizeof(float)) +
                 align_up((size_t)B * sizeof(double)) + align_up(xbits_bytes(T, B, n_in));
    // whole 8-wide runs of inputs and hidden neurons; T <= 32 (the readout's
    // two 16-step row blocks)
    p.ok = p.ok && n_in % 8 == 0 && n_hid % 8 == 0 && n_out <= kFusedMaxOut && T <= 32;
    return p;
}

hipError_t launch_fused_step(const FusedStep &f, void *ws, hipStream_t s) {
    const FusedPlan p = fused_plan(f.T, f.B, f.n_in, f.n_hid, f.n_out);
    if (!p.ok) return hipErrorInvalidValue;
    FusedArgs a{};
    a.T = f.T; a.B = f.B; a.n_in = f.n_in; a.n_hid = f.n_hid; a.n_out = f.n_out;
    a.K = f.n_out / f.P; a.P = f.P;
    a.neuron0 = f.neuron0; a.neuron1 = f.neuron1; a.rs0 = f.rs0; a.rs1 = f.rs1;
    a.alpha0 = f.alpha0; a.beta0 = f.beta0; a.thr0 = f.thr0; a.slope0 = f.slope0;
    a.alpha1 = f.alpha1; a.beta1 = f.beta1; a.thr1 = f.thr1; a.slope1 = f.slope1;
    a.loss_kind = f.loss_kind;
    a.wait_limit = f.wait_limit ? f.wait_limit : kDefaultWaitLimit;
    a.x = f.x; a.W0 = f.W0; a.b0 = f.b0; a.W1 = f.W1; a.b1 = f.b1;
    a.labels = f.labels; a.targets = f.targets;
    a.loss = f.loss; a.counts = f.counts; a.gW0 = f.gW0; a.gb0 = f.gb0; a.gW1 = f.gW1; a.gb1 = f.gb1;
    a.spk = f.spk;
    a.status = f.status;
    const size_t R = (size_t)f.T * f.B;
    char *w = reinterpret_cast<char *>(ws);
    a.s0 = reinterpret_cast<uint8_t *>(w);
    const size_t s0b = align_up(R * hid_stride(f.n_hid));
    a.dI1 = reinterpret_cast<float *>(w + s0b);
    const size_t dib = align_up(R * f.n_out * sizeof(float));
    a.lossb = reinterpret_cast<double *>(w + s0b + dib);
    a.xb = reinterpret_cast<uint8_t *>(w + s0b + dib + align_up((size_t)f.B * sizeof(double)));
    const int slot = p.npw == 4 ? 0 : p.npw == 8 ? 1 : 2;
    void *fn = slot == 0 ? kernel_of<4>() : slot == 1 ? kernel_of<8>() : kernel_of<16>();
    // LDS above the default dynamic limit is opted into once per kernel
    static std::atomic<bool> raised[3];
    if (!raised[slot].load(std::memory_order_acquire)) {
        hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize,
                                           (int)kFusedMaxLds);
        if (e != hipSuccess) return e;
        raised[slot].store(true, std::memory_order_release);
    }
    // A plain launch: the grid (at most one workgroup per compute unit, each
    // within the per-unit limits) is resident at once on an idle device, and
    // the bounded waits end the step if it is not.  A cooperative launch,
    // which guarantees residency, measured about 20 us more per step.
    void *args[] = {&a};
    return hipLaunchKernel(fn, dim3(p.grid), dim3(kThreads), args, (unsigned)p.lds, s);
}

}  // namespace snn
