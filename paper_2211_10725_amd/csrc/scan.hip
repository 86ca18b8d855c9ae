// Neuron time scans for gfx950: forward (eqs. 3-7) and the BPTT reverse scan
// with the fast-sigmoid surrogate (eqs. 8-9).
//
// Layout: every tensor is time-major [T, C] with C = B * n columns, column
// fastest.  One lane owns VEC consecutive columns for all T steps and keeps
// the neuron state in registers; a wave therefore streams 64*VEC contiguous
// floats per step (512 bytes for VEC = 2), fully coalesced.  The inputs of the
// next D steps do not depend on the state, so each lane keeps a ring of D
// prefetched steps in registers to keep enough HBM requests in flight while
// the sequential recurrence runs.
//
// Saved state: the backward needs u_t at every step (the surrogate is a
// function of u_t alone).  Instead of writing u (4 B per step and column) the
// forward writes the state every kCkpt steps (checkpoints: u, and i for the
// current-based neuron), and the reverse scan recomputes each chunk of kCkpt
// steps forward from its checkpoint and the currents, in registers and with
// the forward's exact fp32 operations (so u is bit-identical), before
// running the chunk backwards.
#include <atomic>

#include "neuron.hpp"

namespace snn {
namespace {

constexpr int kThreads = 256;
// Lanes own 2 columns when there are enough columns to fill the chip (2^19:
// 4096 waves of 2-column lanes; on the 65536 x 64-column layer 2 columns and
// 16 steps ahead measured 4-7 % faster than 4 columns and 8 steps, and 1
// column slower still), otherwise 1; the forward loads 16 steps ahead.
constexpr int kWideColumns = 4 * 64 * 2048;
constexpr int kCkpt = kCheckpointInterval;  // steps per recomputed chunk
constexpr int kFoldMax = 16;   // most outputs of a dense layer whose input gradient is folded
constexpr int kFoldRows = 5;   // batch rows one workgroup's columns can span when folding

template <int VEC>
struct Vec;
template <>
struct Vec<2> {
    static __device__ inline void load(const float *p, float (&v)[2]) {
        const float2 x = *reinterpret_cast<const float2 *>(p);
        v[0] = x.x; v[1] = x.y;
    }
    static __device__ inline void store(float *p, const float (&v)[2]) {
        *reinterpret_cast<float2 *>(p) = make_float2(v[0], v[1]);
    }
};
template <>
struct Vec<1> {
    static __device__ inline void load(const float *p, float (&v)[1]) { v[0] = *p; }
    static __device__ inline void store(float *p, const float (&v)[1]) { *p = v[0]; }
};

// spikes as bytes 0/1
template <int VEC>
__device__ inline void store_spikes_u8(uint8_t *p, const float (&z)[VEC]) {
    if constexpr (VEC == 2) {
        *reinterpret_cast<uint16_t *>(p) = (uint16_t)((uint32_t)z[0] | ((uint32_t)z[1] << 8));
    } else {
        p[0] = (uint8_t)z[0];
    }
}

// spikes as fp16 0.0 / 1.0 (0x3c00)
template <int VEC>
__device__ inline void store_spikes_f16(uint16_t *p, const float (&z)[VEC]) {
    if constexpr (VEC == 2) {
        *reinterpret_cast<uint32_t *>(p) =
            (z[0] != 0.f ? 0x3c00u : 0u) | (z[1] != 0.f ? 0x3c000000u : 0u);
    } else {
        p[0] = z[0] != 0.f ? 0x3c00u : 0u;
    }
}

// Spikes packed to bits, one wave's columns per step: a ballot per column
// slot of the lanes.  Lanes that pack bits own the columns w0 + lane + 64 v
// of their wave's 64 VEC columns (w0 the wave's first column, a multiple of
// 64 VEC: the launcher takes VEC = 2 only when C is a multiple of 128, and C
// is a multiple of 64), so ballot v is the 64-bit word of columns
// w0 + 64 v .. + 63.  Lane 0 stores the wave's VEC words.
template <int VEC>
__device__ inline void store_spikes_bits(uint64_t *words, int64_t wave_off, const float (&z)[VEC]) {
    const int lane = threadIdx.x & 63;
    const uint64_t w0 = __ballot(z[0] > 0.f);
    if constexpr (VEC == 2) {
        const uint64_t w1 = __ballot(z[1] > 0.f);
        if (lane == 0)
            *reinterpret_cast<ulonglong2 *>(words + wave_off / 64) = make_ulonglong2(w0, w1);
    } else {
        if (lane == 0) words[wave_off / 64] = w0;
    }
}

// Forward scan.  Writes the spikes, the spike counts (nullable), the full
// membrane (u_out, nullable; it may alias cur exactly: each lane reads step
// t before it writes it) and the checkpoints: after step t with
// (t + 1) % kCkpt == 0 and t + 1 < T, u to ckpt[(t + 1) / kCkpt - 1][C]
// and, for the current-based neuron, i to the same slot of a second plane
// nck chunks further.  The recurrent neuron (eq. 7) adds its own previous
// spike through the recurrent weight: a spike at t-1 adds (v - thr) to u_t
// instead of the plain reset -thr; column c is neuron c % N.
template <int NEURON, int VEC, int OUT, int kDepth>
__global__ __launch_bounds__(kThreads) void neuron_fwd_kernel(int T, int64_t C, int64_t N,
                                                              float alpha, float beta, float thr,
                                                              const float *__restrict__ vrec,
                                                              const float *cur, void *spk,
                                                              float *u_out,
                                                              float *__restrict__ ckpt,
                                                              float *__restrict__ counts) {
    static_assert(kCkpt % kDepth == 0, "checkpoints fall on block boundaries");
    // packed-bit output with two columns per lane: the lane's columns are col
    // and col + 64 (see store_spikes_bits), else col and col + 1
    constexpr bool SPLIT = OUT == SNN_SPK_BITS && VEC == 2;
    constexpr int CS = SPLIT ? 64 : 1;  // column stride within a lane
    const int64_t gid = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    const int64_t col = SPLIT ? (gid >> 6) * 128 + (gid & 63) : gid * VEC;
    if (col >= C) return;
    auto ld = [&](const float *p, float (&v)[VEC]) {
        if constexpr (SPLIT) {
            v[0] = p[0];
            v[1] = p[64];
        } else {
            Vec<VEC>::load(p, v);
        }
    };
    auto st = [&](float *p, const float (&v)[VEC]) {
        if constexpr (SPLIT) {
            p[0] = v[0];
            p[64] = v[1];
        } else {
            Vec<VEC>::store(p, v);
        }
    };
    const int nck = (T - 1) / kCkpt;
    float u[VEC], syn[VEC], zp[VEC], cnt[VEC], jump[VEC];
#pragma unroll
    for (int v = 0; v < VEC; ++v) {
        u[v] = syn[v] = zp[v] = cnt[v] = 0.f;
        if constexpr (NEURON == SNN_RLEAKY) jump[v] = vrec[(col + CS * v) % N] - thr;
        else jump[v] = -thr;
    }

    float in[kDepth][VEC], nx[kDepth][VEC];
#pragma unroll
    for (int j = 0; j < kDepth; ++j)
        if (j < T) ld(cur + (int64_t)j * C + col, in[j]);

    for (int t0 = 0; t0 < T; t0 += kDepth) {
#pragma unroll
        for (int j = 0; j < kDepth; ++j)
            if (t0 + kDepth + j < T) ld(cur + (int64_t)(t0 + kDepth + j) * C + col, nx[j]);
#pragma unroll
        for (int j = 0; j < kDepth; ++j) {
            const int t = t0 + j;
            if (t < T) {
                float z[VEC];
#pragma unroll
                for (int v = 0; v < VEC; ++v) {
                    const float uu = neuron_step<NEURON>(u[v], syn[v], zp[v], in[j][v], alpha,
                                                         beta, jump[v]);
                    z[v] = (uu > thr) ? 1.f : 0.f;       // eq. (3), strict
                    zp[v] = z[v];
                    cnt[v] += z[v];
                }
                const int64_t off = (int64_t)t * C + col;
                if (u_out) st(u_out + off, u);
                if constexpr (OUT == SNN_U8)
                    store_spikes_u8<VEC>(reinterpret_cast<uint8_t *>(spk) + off, z);
                else if constexpr (OUT == SNN_SPK_BITS)
                    store_spikes_bits<VEC>(reinterpret_cast<uint64_t *>(spk),
                                           off - (threadIdx.x & 63), z);
                else
                    store_spikes_f16<VEC>(reinterpret_cast<uint16_t *>(spk) + off, z);
            }
        }
        const int tn = t0 + kDepth;  // steps done
        if (tn % kCkpt == 0 && tn < T) {
            const int64_t slot = (int64_t)(tn / kCkpt - 1) * C + col;
            st(ckpt + slot, u);
            if constexpr (NEURON == SNN_SYNAPTIC) st(ckpt + (int64_t)nck * C + slot, syn);
        }
#pragma unroll
        for (int j = 0; j < kDepth; ++j)
#pragma unroll
            for (int v = 0; v < VEC; ++v) in[j][v] = nx[j][v];
    }
    if (counts) st(counts + col, cnt);
}

__device__ inline uint16_t f32_to_bf16_rne(float x) {
    const uint32_t b = __float_as_uint(x);
    return (uint16_t)((b + 0x7fffu + ((b >> 16) & 1u)) >> 16);
}

// dL/dI in the operand type of the contractions.  fp16 is written scaled by
// the power of two `scale` (exact), chosen per call so that every value
// stays below 2^15 (grad_scale_*_kernel below).
template <int GT, int VEC>
__device__ inline void store_grad(void *base, int64_t off, const float (&v)[VEC], float scale) {
    if constexpr (GT == SNN_F32) {
        Vec<VEC>::store(reinterpret_cast<float *>(base) + off, v);
    } else {
        uint16_t h[VEC];
#pragma unroll
        for (int i = 0; i < VEC; ++i) {
            if constexpr (GT == SNN_F16) {
                const _Float16 f = (_Float16)(v[i] * scale);
                h[i] = __builtin_bit_cast(uint16_t, f);
            } else {
                h[i] = f32_to_bf16_rne(v[i]);
            }
        }
        uint16_t *p = reinterpret_cast<uint16_t *>(base) + off;
        if constexpr (VEC == 2)
            *reinterpret_cast<uint32_t *>(p) = (uint32_t)h[0] | ((uint32_t)h[1] << 16);
        else
            p[0] = h[0];
    }
}

// The 16-bit parts of dL/dI for the weight-gradient contraction: fp32 as
// three exact bf16 parts (hi = bf16(x), mid = bf16(x - hi), lo = bf16(x - hi
// - mid), each subtraction exact), bf16 or fp16 (scaled) as one.
__device__ inline uint32_t bf16_rne_bits(float x) { return f32_to_bf16_rne(x); }
template <int GT>
__device__ inline uint32_t grad_part(float x, int p, float scale) {
    if constexpr (GT == SNN_F16) {
        const _Float16 f = (_Float16)(x * scale);
        return __builtin_bit_cast(uint16_t, f);
    } else if constexpr (GT == SNN_BF16) {
        return bf16_rne_bits(x);
    } else {
        const uint32_t hi = bf16_rne_bits(x);
        if (p == 0) return hi;
        const float r = x - __uint_as_float(hi << 16);
        const uint32_t mid = bf16_rne_bits(r);
        if (p == 1) return mid;
        return bf16_rne_bits(r - __uint_as_float(mid << 16));
    }
}

// Sources of the upstream gradient g_t = dL/dz_t of the reverse scan.
constexpr int GM_FULL = 0;   // g [T, C]
constexpr int GM_BCAST = 1;  // g [C], the same for every t
constexpr int GM_FOLD = 2;   // g_t[b, n] = sum_j dI_up[t, b, j] W_up[j, n]: the input
                             // gradient of a dense layer above with at most
                             // kFoldMax outputs, computed here instead of read
constexpr int GM_FOLD12 = 3; // the same for at most 12 outputs (10 classes)

// The layer above, for GM_FOLD.  A workgroup's 256 VEC consecutive columns
// span at most kFoldRows batch rows (the launcher only folds layers with
// n >= 64, and n >= 128 for VEC = 2); the dI_up rows of those batch rows for
// one chunk of kCkpt steps are staged in LDS (double-buffered, one barrier
// per chunk), the next chunk's loaded into registers while this one runs.
struct FoldIn {
    const void *dup;  // [T, B, nup] of dt_up
    const void *wup;  // [nup, N] of dt_w
    int nup, dt_up, dt_w, B;
};

__device__ inline float load_as_f32(const void *p, int64_t i, int dt) {
    if (dt == SNN_F32) return reinterpret_cast<const float *>(p)[i];
    const uint16_t h = reinterpret_cast<const uint16_t *>(p)[i];
    if (dt == SNN_BF16) return __uint_as_float((uint32_t)h << 16);
    return (float)__builtin_bit_cast(_Float16, h);
}

template <int KF>
struct FoldStage {
    static constexpr int kElems = kCkpt * kFoldRows * KF;
    static constexpr int kPer = (kElems + 255) / 256;  // per thread (256-thread blocks)
    float v[kPer];

    // the dI_up values of the steps t0 .. t0 + kCkpt - 1 of a chunk and batch
    // rows b_lo .. b_lo + kFoldRows - 1 (zeros outside)
    __device__ inline void load(const FoldIn &f, int T, int t0, int64_t b_lo) {
#pragma unroll
        for (int i = 0; i < kPer; ++i) {
            const int e = threadIdx.x + i * 256;
            const int jt = e / (kFoldRows * KF), bb = (e / KF) % kFoldRows, j = e % KF;
            const int t = t0 + jt;
            const int64_t b = b_lo + bb;
            v[i] = (e < kElems && t < T && b < f.B && j < f.nup)
                       ? load_as_f32(f.dup, ((int64_t)t * f.B + b) * f.nup + j, f.dt_up)
                       : 0.f;
        }
    }
    __device__ inline void store(float *rows) const {
#pragma unroll
        for (int i = 0; i < kPer; ++i) {
            const int e = threadIdx.x + i * 256;
            if (e < kElems) rows[e] = v[i];
        }
    }
};

// Reverse-time scan over chunks of kCkpt steps, last chunk first.  For each
// chunk the lane loads its currents and the checkpoint before it (prefetched
// while the previous chunk runs), recomputes u_t forward in registers, then
// runs the adjoint backwards.  lam carries dL/du_{t+1} (and lami dL/di_{t+1}).
// For the recurrent neuron the spike z_t reaches u_{t+1} through
// (v - r thr), so the carry is beta + (v - r thr) s_t, and the recurrent
// weight's gradient collects lam_{t+1} z_t per column (dvcol, fp32).
//
// With TR = TR_TRANSPOSED, dL/dI is also written as the weight gradient's
// operand: dcur_t [P][N][B*T] (P = 3 bf16 parts of fp32, else 1 plane of the
// 16-bit type, planes t_plane elements apart), row n holding column n of
// every sample, K index b*T + t.  A lane's column is one row there and a
// chunk's steps are consecutive in it, so each chunk's values are packed in
// registers as the reverse loop produces them and stored together.  With
// TR = TR_PLANES (fp32 only), dcur_t holds the three bf16 parts in dcur's own
// layout, [3][T][C], written at every step like dcur.  The row-major dcur
// may be skipped (nullptr) in both cases.
constexpr int TR_NONE = 0, TR_TRANSPOSED = 1, TR_PLANES = 2;
template <int NEURON, int VEC, int GM, bool RESET_SURR, int GT, int TRM>
__global__ __launch_bounds__(kThreads) void neuron_bwd_kernel(
    int T, int64_t C, int64_t N, float alpha, float beta, float thr, float slope,
    const float *__restrict__ vrec, const float *__restrict__ cur, const float *__restrict__ ckpt,
    const float *__restrict__ g, FoldIn fold, void *__restrict__ dcur,
    uint16_t *__restrict__ dcur_t, int64_t t_plane,
    const float *__restrict__ dscale, float *__restrict__ colsum, float *__restrict__ dvcol) {
    constexpr bool BCAST = GM == GM_BCAST, FOLD = GM == GM_FOLD || GM == GM_FOLD12;
    constexpr bool FULL = GM == GM_FULL;
    constexpr int K = kCkpt;
    constexpr int P = GT == SNN_F32 ? 3 : 1;  // 16-bit parts per value in dcur_t
    constexpr bool TR = TRM == TR_TRANSPOSED;
    uint32_t pk[TR ? P : 1][TR ? VEC : 1][TR ? K / 2 : 1];  // packed parts of a chunk
    const float scale = GT == SNN_F16 ? *dscale : 1.f;
    constexpr int KF = GM == GM_FOLD12 ? 12 : kFoldMax;  // dI_up values per row (padded)
    const int64_t col = ((int64_t)blockIdx.x * kThreads + threadIdx.x) * VEC;
    // the fold's lanes past the last column still take part in the staging
    const bool active = col < C;
    if (!FOLD && !active) return;
    const int nch = (T + K - 1) / K, nck = nch - 1;
    float lam[VEC], lami[VEC], acc[VEC], gb[VEC], vr[VEC], dv[VEC], jump[VEC];
#pragma unroll
    for (int v = 0; v < VEC; ++v) {
        lam[v] = lami[v] = acc[v] = gb[v] = dv[v] = 0.f;
        const float vv = (NEURON == SNN_RLEAKY && active) ? vrec[(col + v) % N] : 0.f;
        jump[v] = NEURON == SNN_RLEAKY ? vv - thr : -thr;
        vr[v] = NEURON == SNN_RLEAKY ? (RESET_SURR ? vv - thr : vv) : 0.f;
    }
    if constexpr (BCAST) Vec<VEC>::load(g + col, gb);

    // fold: the lane's columns of W_up, its batch row within the staged rows
    __shared__ __attribute__((aligned(16))) float frows[FOLD ? 2 : 1][FOLD ? FoldStage<KF>::kElems : 1];
    float wcol[FOLD ? VEC : 1][FOLD ? KF : 1];
    int fbb = 0;
    int64_t b_lo = 0;
    FoldStage<KF> fst;
    if constexpr (FOLD) {
        b_lo = ((int64_t)blockIdx.x * kThreads * VEC) / N;
        fbb = active ? (int)(col / N - b_lo) : 0;
#pragma unroll
        for (int v = 0; v < VEC; ++v)
#pragma unroll
            for (int j = 0; j < KF; ++j)
                wcol[v][j] = (active && j < fold.nup)
                                 ? load_as_f32(fold.wup, (int64_t)j * N + (col + v) % N, fold.dt_w)
                                 : 0.f;
        fst.load(fold, T, nck * K, b_lo);
        fst.store(frows[nck & 1]);
        if (nck >= 1) fst.load(fold, T, (nck - 1) * K, b_lo);
        __syncthreads();
    }

    // chunk registers: currents (then the recomputed membrane) of this chunk
    // and of the one before it, the full upstream gradient likewise, and the
    // checkpointed state at the start of each
    float ii[K][VEC], ni[K][VEC];
    float gg[FULL ? K : 1][VEC], ng[FULL ? K : 1][VEC];
    float cu[VEC], ci[VEC], nu[VEC], nci[VEC];
    auto load_chunk = [&](int c, float (&xi)[K][VEC], float (&xg)[FULL ? K : 1][VEC],
                          float (&su)[VEC], float (&si)[VEC]) {
        const int t_lo = c * K;
#pragma unroll
        for (int j = 0; j < K; ++j) {
            if (t_lo + j < T) {
                Vec<VEC>::load(cur + (int64_t)(t_lo + j) * C + col, xi[j]);
                if constexpr (FULL) Vec<VEC>::load(g + (int64_t)(t_lo + j) * C + col, xg[j]);
            }
        }
        if (c > 0) {
            Vec<VEC>::load(ckpt + (int64_t)(c - 1) * C + col, su);
            if constexpr (NEURON == SNN_SYNAPTIC)
                Vec<VEC>::load(ckpt + (int64_t)(nck + c - 1) * C + col, si);
            else
#pragma unroll
                for (int v = 0; v < VEC; ++v) si[v] = 0.f;
        } else {
#pragma unroll
            for (int v = 0; v < VEC; ++v) su[v] = si[v] = 0.f;
        }
    };
    if (active) load_chunk(nck, ii, gg, cu, ci);

    for (int c = nck; c >= 0; --c) {
        const int t_lo = c * K;
        if (active) {
            if (c > 0) load_chunk(c - 1, ni, ng, nu, nci);
            // recompute u_t of the chunk from the state before it (u_{t_lo-1},
            // i_{t_lo-1}; z_{t_lo-1} = [u_{t_lo-1} > thr]), in place of I_t
#pragma unroll
            for (int v = 0; v < VEC; ++v) {
                float u = cu[v], syn = ci[v];
                float zp = (c > 0 && cu[v] > thr) ? 1.f : 0.f;
#pragma unroll
                for (int j = 0; j < K; ++j) {
                    if (t_lo + j < T) {
                        const float uu = neuron_step<NEURON>(u, syn, zp, ii[j][v], alpha, beta,
                                                             jump[v]);
                        ii[j][v] = uu;
                        zp = (uu > thr) ? 1.f : 0.f;
                    }
                }
            }
        }
        const float *fr = FOLD ? frows[c & 1] : nullptr;
        if constexpr (TR) {
#pragma unroll
            for (int p = 0; p < P; ++p)
#pragma unroll
                for (int v = 0; v < VEC; ++v)
#pragma unroll
                    for (int q = 0; q < K / 2; ++q) pk[p][v][q] = 0u;
        }
#pragma unroll
        for (int j = K - 1; j >= 0; --j) {
            const int t = t_lo + j;
            if (t < T && active) {
                float d[VEC];
                float grow[FOLD ? KF : 1];
                if constexpr (FOLD) {
                    const float4 *r4 = reinterpret_cast<const float4 *>(
                        fr + (j * kFoldRows + fbb) * KF);
#pragma unroll
                    for (int q = 0; q < KF / 4; ++q) {
                        const float4 x = r4[q];
                        grow[4 * q] = x.x; grow[4 * q + 1] = x.y;
                        grow[4 * q + 2] = x.z; grow[4 * q + 3] = x.w;
                    }
                }
#pragma unroll
                for (int v = 0; v < VEC; ++v) {
                    const float uu = ii[j][v];
                    const float s = surrogate(uu, thr, slope);
                    float gt;
                    if constexpr (BCAST) {
                        gt = gb[v];
                    } else if constexpr (FOLD) {
                        gt = 0.f;  // j ascending: the order of the short contraction
#pragma unroll
                        for (int q = 0; q < KF; ++q) gt = __builtin_fmaf(grow[q], wcol[v][q], gt);
                    } else {
                        gt = gg[j][v];
                    }
                    if constexpr (NEURON == SNN_RLEAKY) {
                        if (uu > thr) dv[v] += lam[v];  // lam_{t+1} z_t
                        const float carry = __builtin_fmaf(vr[v], s, beta);
                        lam[v] = __builtin_fmaf(carry, lam[v], gt * s);
                        d[v] = lam[v];
                    } else {
                        d[v] = adjoint_step<NEURON, RESET_SURR>(lam[v], lami[v], gt, s, alpha,
                                                                beta, thr);
                    }
                    acc[v] += d[v];
                }
                if (dcur) store_grad<GT, VEC>(dcur, (int64_t)t * C + col, d, scale);
                if constexpr (TRM == TR_PLANES) {
#pragma unroll
                    for (int p = 0; p < 3; ++p) {
                        uint16_t *q = dcur_t + p * t_plane + (int64_t)t * C + col;
                        const uint32_t h0 = grad_part<SNN_F32>(d[0], p, 1.f);
                        if constexpr (VEC == 2)
                            *reinterpret_cast<uint32_t *>(q) = h0 | (grad_part<SNN_F32>(d[1], p, 1.f) << 16);
                        else
                            q[0] = (uint16_t)h0;
                    }
                }
                if constexpr (TR) {
#pragma unroll
                    for (int p = 0; p < P; ++p)
#pragma unroll
                        for (int v = 0; v < VEC; ++v) {
                            const uint32_t h = grad_part<GT>(d[v], p, scale);
                            pk[p][v][j / 2] |= (j & 1) ? h << 16 : h;
                        }
                }
            }
        }
        if constexpr (TR) {
            // the chunk's steps of this lane's columns, row (col + v) % N,
            // K index b*T + t
            if (active) {
                const int len = min(K, T - t_lo);
#pragma unroll
                for (int v = 0; v < VEC; ++v) {
                    const int64_t n = (col + v) % N, b = (col + v) / N;
                    const int64_t base = n * ((int64_t)T * (C / N)) + b * T + t_lo;
#pragma unroll
                    for (int p = 0; p < P; ++p) {
                        uint16_t *row = dcur_t + p * t_plane + base;
                        if (len == K && (T & 3) == 0) {
#pragma unroll
                            for (int q = 0; q < K / 4; ++q)
                                *reinterpret_cast<uint2 *>(row + 4 * q) =
                                    make_uint2(pk[p][v][2 * q], pk[p][v][2 * q + 1]);
                        } else {
#pragma unroll
                            for (int jj = 0; jj < K; ++jj)
                                if (jj < len)
                                    row[jj] = (uint16_t)(pk[p][v][jj / 2] >> (16 * (jj & 1)));
                        }
                    }
                }
            }
        }
        if constexpr (FOLD) {
            // stage the next chunk (its buffer was last read before the
            // previous barrier), then load the one after it
            if (c >= 1) {
                fst.store(frows[(c - 1) & 1]);
                if (c >= 2) fst.load(fold, T, (c - 2) * K, b_lo);
            }
            __syncthreads();
        }
#pragma unroll
        for (int j = 0; j < K; ++j)
#pragma unroll
            for (int v = 0; v < VEC; ++v) {
                ii[j][v] = ni[j][v];
                if constexpr (FULL) gg[j][v] = ng[j][v];
            }
#pragma unroll
        for (int v = 0; v < VEC; ++v) {
            cu[v] = nu[v];
            ci[v] = nci[v];
        }
    }
    if (!active) return;
    if (colsum) Vec<VEC>::store(colsum + col, acc);
    if constexpr (NEURON == SNN_RLEAKY)
        if (dvcol) Vec<VEC>::store(dvcol + col, dv);
}

// Bias gradient: db[f] = sum over b of the per-column time sums.  A block
// owns 64 consecutive features (one per lane); its 16 waves take every 16th
// batch row, each lane summing in fp64 in a fixed order, and the 16 partial
// sums are added in wave order.
__global__ __launch_bounds__(1024) void bias_reduce_kernel(int B, int F,
                                                           const float *__restrict__ colsum,
                                                           float *__restrict__ db) {
    __shared__ double part[16][64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int f = blockIdx.x * 64 + lane;
    double acc = 0.0;
    if (f < F) {
#pragma unroll 4
        for (int b = wave; b < B; b += 16) acc += (double)colsum[(int64_t)b * F + f];
    }
    part[wave][lane] = acc;
    __syncthreads();
    if (wave == 0 && f < F) {
        double s = 0.0;
#pragma unroll
        for (int w = 0; w < 16; ++w) s += part[w][lane];
        db[f] = (float)s;
    }
}

// The same sum for layers with P > 1 positions per feature (conv channels):
// one 1024-thread block per feature, fp64 partial sums over a fixed
// assignment of (b, p) to threads, then a fixed-order tree.
constexpr int kReduceThreads = 1024;
__global__ __launch_bounds__(kReduceThreads) void bias_reduce_pos_kernel(
    int B, int F, int P, const float *__restrict__ colsum, float *__restrict__ db) {
    __shared__ double part[kReduceThreads];
    const int f = blockIdx.x;
    const int64_t n = (int64_t)B * P;
    double acc = 0.0;
    for (int64_t j = threadIdx.x; j < n; j += kReduceThreads)
        acc += (double)colsum[((j / P) * F + f) * P + j % P];
    part[threadIdx.x] = acc;
    __syncthreads();
    for (int w = kReduceThreads / 2; w > 0; w >>= 1) {
        if ((int)threadIdx.x < w) part[threadIdx.x] += part[threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x == 0) db[f] = (float)part[0];
}

// ---- the power-of-two scale of an fp16 dL/dI ------------------------------
// |lam_t| <= G F with G a bound on |g| and F = sum_k c^k the growth of the
// reverse recursion (computed by the caller from beta, alpha, thr and T), so
// dL/dI S with S = 2^e, e = floor(log2(2^15 / (G F))), stays below 2^15
// (fp16 holds up to 65504: a factor 2 of headroom for the fp32 rounding of
// the bound and the recursion).  G is a max over the upstream gradient:
//   FULL / BCAST  G = max |g|
//   FOLD          G = max_{t,b} sum_j |dup[t,b,j]|  *  max_{j,n} |wup[j,n]|
//                 (>= |sum_j dup[t,b,j] wup[j,n]| for every n)
// First pass: per-workgroup maxima (partial[2 blk], partial[2 blk + 1]);
// second pass, one workgroup: the maxima, G and S (written to scale[0]).
// Max is order-independent: the result is deterministic.
constexpr int kScaleBlocks = 1024;

__device__ inline float block_max(float v, float *red) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (lane == 0) red[wave] = v;
    __syncthreads();
    float m = 0.f;
    for (int w = 0; w < (int)(blockDim.x >> 6); ++w) m = fmaxf(m, red[w]);
    __syncthreads();
    return m;
}

__global__ __launch_bounds__(kThreads) void grad_bound_kernel(int64_t rows, int width, int dt,
                                                              const void *__restrict__ src,
                                                              int64_t nw, int dt_w,
                                                              const void *__restrict__ w,
                                                              float *__restrict__ partial) {
    __shared__ float red[kThreads / 64];
    // rows of `width` values: the max over rows of sum |x| (width 1: max |x|)
    float m1 = 0.f;
    for (int64_t r = (int64_t)blockIdx.x * kThreads + threadIdx.x; r < rows;
         r += (int64_t)gridDim.x * kThreads) {
        float a = 0.f;
        for (int j = 0; j < width; ++j) a += __builtin_fabsf(load_as_f32(src, r * width + j, dt));
        m1 = fmaxf(m1, a);
    }
    float m2 = 0.f;
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < nw;
         i += (int64_t)gridDim.x * kThreads)
        m2 = fmaxf(m2, __builtin_fabsf(load_as_f32(w, i, dt_w)));
    m1 = block_max(m1, red);
    m2 = block_max(m2, red);
    if (threadIdx.x == 0) {
        partial[2 * blockIdx.x] = m1;
        partial[2 * blockIdx.x + 1] = m2;
    }
}

__global__ __launch_bounds__(kThreads) void grad_scale_kernel(int nblk, bool product, double growth,
                                                              const float *__restrict__ partial,
                                                              float *__restrict__ scale) {
    __shared__ float red[kThreads / 64];
    float m1 = 0.f, m2 = 0.f;
    for (int i = threadIdx.x; i < nblk; i += kThreads) {
        m1 = fmaxf(m1, partial[2 * i]);
        m2 = fmaxf(m2, partial[2 * i + 1]);
    }
    m1 = block_max(m1, red);
    m2 = block_max(m2, red);
    if (threadIdx.x == 0) {
        const double G = product ? (double)m1 * (double)m2 : (double)m1;
        const double bound = G * growth;
        int e = 0;
        if (bound > 0.0 && bound < 1e300) {
            int ex;
            (void)frexp(32768.0 / bound, &ex);  // 32768 / bound in [2^(ex-1), 2^ex)
            e = ex - 1;
            if (e > 120) e = 120;
            if (e < -120) e = -120;
        }
        scale[0] = ldexpf(1.f, e);
    }
}

__global__ __launch_bounds__(kThreads) void fill_zero_kernel(float *__restrict__ p, int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (i < n) p[i] = 0.f;
}

struct ScanArgs {
    int T;
    int64_t C, N;
    float alpha, beta, thr, slope;
    const float *vrec;
};

struct FwdBuffers {
    const float *cur;
    void *spk;
    float *u_out, *ckpt, *counts;
};

template <int NEURON, int VEC, int OUT>
void fwd_launch(const ScanArgs &a, const FwdBuffers &b, hipStream_t s) {
    const int64_t lanes = (a.C + VEC - 1) / VEC;
    const unsigned grid = (unsigned)((lanes + kThreads - 1) / kThreads);
    neuron_fwd_kernel<NEURON, VEC, OUT, 16><<<grid, kThreads, 0, s>>>(
        a.T, a.C, a.N, a.alpha, a.beta, a.thr, a.vrec, b.cur, b.spk, b.u_out, b.ckpt, b.counts);
}

template <int NEURON, int VEC>
void fwd_dispatch(int out_dtype, const ScanArgs &a, const FwdBuffers &b, hipStream_t s) {
    if (out_dtype == SNN_U8) fwd_launch<NEURON, VEC, SNN_U8>(a, b, s);
    else if (out_dtype == SNN_SPK_BITS) fwd_launch<NEURON, VEC, SNN_SPK_BITS>(a, b, s);
    else fwd_launch<NEURON, VEC, SNN_F16>(a, b, s);
}

struct BwdBuffers {
    const float *cur, *ckpt, *g;
    FoldIn fold;
    void *dcur;
    uint16_t *dcur_t;
    bool planes;  // dcur_t holds the planes of an fp32 dL/dI in dcur's layout
    const float *dscale;
    float *colsum, *dvcol;
};

template <int NEURON, int VEC, int GM, bool RS, int GT>
void bwd_launch(const ScanArgs &a, const BwdBuffers &b, hipStream_t s) {
    const int64_t lanes = (a.C + VEC - 1) / VEC;
    const unsigned grid = (unsigned)((lanes + kThreads - 1) / kThreads);
    const int64_t t_plane = (int64_t)a.T * a.C;
    if (b.dcur_t && b.planes) {
        if constexpr (GT == SNN_F32)
            neuron_bwd_kernel<NEURON, VEC, GM, RS, GT, TR_PLANES><<<grid, kThreads, 0, s>>>(
                a.T, a.C, a.N, a.alpha, a.beta, a.thr, a.slope, a.vrec, b.cur, b.ckpt, b.g,
                b.fold, b.dcur, b.dcur_t, t_plane, b.dscale, b.colsum, b.dvcol);
    } else if (b.dcur_t) {
        neuron_bwd_kernel<NEURON, VEC, GM, RS, GT, TR_TRANSPOSED><<<grid, kThreads, 0, s>>>(
            a.T, a.C, a.N, a.alpha, a.beta, a.thr, a.slope, a.vrec, b.cur, b.ckpt, b.g, b.fold,
            b.dcur, b.dcur_t, t_plane, b.dscale, b.colsum, b.dvcol);
    } else {
        neuron_bwd_kernel<NEURON, VEC, GM, RS, GT, TR_NONE><<<grid, kThreads, 0, s>>>(
            a.T, a.C, a.N, a.alpha, a.beta, a.thr, a.slope, a.vrec, b.cur, b.ckpt, b.g, b.fold,
            b.dcur, nullptr, 0, b.dscale, b.colsum, b.dvcol);
    }
}

template <int NEURON, int VEC, int GM, bool RS>
void bwd_dispatch_gt(int gt, const ScanArgs &a, const BwdBuffers &b, hipStream_t s) {
    if (gt == SNN_F32) bwd_launch<NEURON, VEC, GM, RS, SNN_F32>(a, b, s);
    else if (gt == SNN_F16) bwd_launch<NEURON, VEC, GM, RS, SNN_F16>(a, b, s);
    else bwd_launch<NEURON, VEC, GM, RS, SNN_BF16>(a, b, s);
}

template <int NEURON, int VEC, int GM>
void bwd_dispatch_rs(int rs, int gt, const ScanArgs &a, const BwdBuffers &b, hipStream_t s) {
    if (rs) bwd_dispatch_gt<NEURON, VEC, GM, true>(gt, a, b, s);
    else bwd_dispatch_gt<NEURON, VEC, GM, false>(gt, a, b, s);
}

// Lane widths: two columns for layers of at least kWideColumns columns
// (measured on the 65536 x 64-column layer: 7.0 against 7.4 ms for four
// columns per lane, whose chunk registers left two waves per SIMD), else one.
template <int NEURON>
void bwd_dispatch(int vec, int rs, int gm, int gt, const ScanArgs &a, const BwdBuffers &b,
                  hipStream_t s) {
    if (gm == GM_BCAST) {
        if (vec == 2) bwd_dispatch_rs<NEURON, 2, GM_BCAST>(rs, gt, a, b, s);
        else bwd_dispatch_rs<NEURON, 1, GM_BCAST>(rs, gt, a, b, s);
    } else if (gm == GM_FOLD12) {
        if (vec == 2) bwd_dispatch_rs<NEURON, 2, GM_FOLD12>(rs, gt, a, b, s);
        else bwd_dispatch_rs<NEURON, 1, GM_FOLD12>(rs, gt, a, b, s);
    } else if (gm == GM_FOLD) {
        if (vec == 2) bwd_dispatch_rs<NEURON, 2, GM_FOLD>(rs, gt, a, b, s);
        else bwd_dispatch_rs<NEURON, 1, GM_FOLD>(rs, gt, a, b, s);
    } else {
        if (vec == 2) bwd_dispatch_rs<NEURON, 2, GM_FULL>(rs, gt, a, b, s);
        else bwd_dispatch_rs<NEURON, 1, GM_FULL>(rs, gt, a, b, s);
    }
}

}  // namespace

int64_t neuron_ckpt_count(int T) { return T > 0 ? (T - 1) / kCkpt : 0; }

hipError_t launch_neuron_fwd(int neuron, int T, int64_t C, int64_t N, float alpha, float beta,
                             float thr, const float *vrec, const float *cur, void *spk,
                             int out_dtype, float *u_out, float *ckpt, float *counts,
                             hipStream_t s) {
    if (T <= 0 || C <= 0) return hipSuccess;
    if (neuron_ckpt_count(T) > 0 && ckpt == nullptr) return hipErrorInvalidValue;
    // packed spikes: whole 64-bit words per wave (C a multiple of 64 * VEC)
    if (out_dtype == SNN_SPK_BITS && C % 64 != 0) return hipErrorInvalidValue;
    const bool v2 = (C % 2) == 0 && C >= kWideColumns && (out_dtype != SNN_SPK_BITS || C % 128 == 0);
    const ScanArgs a{T, C, N, alpha, beta, thr, 0.f, vrec};
    const FwdBuffers b{cur, spk, u_out, ckpt, counts};
    switch (neuron) {
        case SNN_SYNAPTIC:
            if (v2) fwd_dispatch<SNN_SYNAPTIC, 2>(out_dtype, a, b, s);
            else fwd_dispatch<SNN_SYNAPTIC, 1>(out_dtype, a, b, s);
            break;
        case SNN_RLEAKY:
            if (v2) fwd_dispatch<SNN_RLEAKY, 2>(out_dtype, a, b, s);
            else fwd_dispatch<SNN_RLEAKY, 1>(out_dtype, a, b, s);
            break;
        default:
            if (v2) fwd_dispatch<SNN_LEAKY, 2>(out_dtype, a, b, s);
            else fwd_dispatch<SNN_LEAKY, 1>(out_dtype, a, b, s);
    }
    return hipGetLastError();
}

bool neuron_fold_supported(int64_t N) { return N >= 64; }

hipError_t launch_neuron_bwd(int neuron, int reset_surrogate, int T, int64_t C, int64_t N,
                             float alpha, float beta, float thr, float slope, const float *vrec,
                             const float *cur, const float *ckpt, const BwdGrad &grad, int B,
                             void *dcur, void *dcur_t, bool dcur_t_planes, int grad_dtype,
                             const float *dscale, float *colsum, float *dvcol, hipStream_t s) {
    if (dcur == nullptr && dcur_t == nullptr) return hipErrorInvalidValue;
    if (dcur_t && dcur_t_planes && grad_dtype != SNN_F32) return hipErrorInvalidValue;
    if (grad_dtype == SNN_F16 && dscale == nullptr) return hipErrorInvalidValue;
    if (T <= 0 || C <= 0) return hipSuccess;
    if (neuron_ckpt_count(T) > 0 && ckpt == nullptr) return hipErrorInvalidValue;
    int gm = grad.mode == SNN_GRAD_FOLD ? GM_FOLD
             : grad.mode == SNN_GRAD_BCAST ? GM_BCAST : GM_FULL;
    if (gm == GM_FOLD && (!neuron_fold_supported(N) || grad.nup < 1 || grad.nup > kFoldMax))
        return hipErrorInvalidValue;
    if (gm == GM_FOLD && grad.nup <= 12) gm = GM_FOLD12;
    const bool wide = C >= kWideColumns;
    int vec = 1;
    if (gm == GM_FULL) {
        if (wide && C % 2 == 0) vec = 2;
    } else if (gm == GM_BCAST) {
        if (wide && C % 2 == 0) vec = 2;
    } else if (wide && N % 2 == 0 && N >= 128) {
        // a lane's two columns in one batch row, and the workgroup's 512
        // columns within kFoldRows batch rows
        vec = 2;
    }
    const ScanArgs a{T, C, N, alpha, beta, thr, slope, vrec};
    const FoldIn fold{grad.dup, grad.wup, grad.nup, grad.dt_up, grad.dt_w, B};
    const BwdBuffers b{cur,  ckpt, grad.g, fold, dcur, reinterpret_cast<uint16_t *>(dcur_t),
                       dcur_t_planes, dscale, colsum, dvcol};
    const int rs = reset_surrogate, gt = grad_dtype;
    switch (neuron) {
        case SNN_SYNAPTIC: bwd_dispatch<SNN_SYNAPTIC>(vec, rs, gm, gt, a, b, s); break;
        case SNN_RLEAKY: bwd_dispatch<SNN_RLEAKY>(vec, rs, gm, gt, a, b, s); break;
        default: bwd_dispatch<SNN_LEAKY>(vec, rs, gm, gt, a, b, s);
    }
    return hipGetLastError();
}

hipError_t launch_fill_zero(float *p, int64_t n, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    fill_zero_kernel<<<(unsigned)((n + kThreads - 1) / kThreads), kThreads, 0, s>>>(p, n);
    return hipGetLastError();
}

size_t grad_scale_workspace_bytes() { return 2 * kScaleBlocks * sizeof(float); }

hipError_t launch_grad_scale(int T, int64_t C, const BwdGrad &grad, int B, double growth,
                             float *scale, float *scratch, hipStream_t s) {
    int64_t rows, nw = 0;
    int width = 1, dt = SNN_F32, dt_w = SNN_F32;
    const void *src, *w = nullptr;
    if (grad.mode == SNN_GRAD_FOLD) {
        rows = (int64_t)T * B;
        width = grad.nup;
        dt = grad.dt_up;
        src = grad.dup;
        nw = (int64_t)grad.nup * (C / B);
        w = grad.wup;
        dt_w = grad.dt_w;
    } else {
        rows = grad.mode == SNN_GRAD_BCAST ? C : (int64_t)T * C;
        src = grad.g;
    }
    const int64_t work = rows * width > nw ? rows * width : nw;
    int nblk = (int)((work + 16 * kThreads - 1) / (16 * kThreads));
    if (nblk < 1) nblk = 1;
    if (nblk > kScaleBlocks) nblk = kScaleBlocks;
    grad_bound_kernel<<<nblk, kThreads, 0, s>>>(rows, width, dt, src, nw, dt_w, w, scratch);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    grad_scale_kernel<<<1, kThreads, 0, s>>>(nblk, grad.mode == SNN_GRAD_FOLD, growth, scratch,
                                             scale);
    return hipGetLastError();
}

int device_cus() {
    static std::atomic<int> cache[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    int v = cache[dev].load(std::memory_order_relaxed);
    if (v == 0) {
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            v <= 0)
            v = 256;
        cache[dev].store(v, std::memory_order_relaxed);
    }
    return v;
}

hipError_t launch_bias_reduce(int B, int F, int P, const float *colsum, float *db, hipStream_t s) {
    if (F <= 0) return hipSuccess;
    if (P > 1) bias_reduce_pos_kernel<<<F, kReduceThreads, 0, s>>>(B, F, P, colsum, db);
    else bias_reduce_kernel<<<(F + 63) / 64, 1024, 0, s>>>(B, F, colsum, db);
    return hipGetLastError();
}

}  // namespace snn
