// Per-column neuron arithmetic shared by the time scans and the fused
// small-batch step: the forward recurrence (eqs. 3-7) and the adjoint
// recursion of BPTT with the fast-sigmoid surrogate (eqs. 8-9), in the exact
// fp32 operations every kernel uses, so all of them give the same bits.
#pragma once

#include "snn_internal.hpp"

namespace snn {

// One step of the forward recurrence for one column: the decay-plus-input
// term as one fused multiply-add (for the current-based neuron, eq. (5)
// first), then the reset jump (-thr, or v - thr for the recurrent neuron of
// eq. (7)) if the previous step spiked.  Returns the new membrane; the spike
// is u > thr (eq. (3), strict).
template <int NEURON>
__device__ inline float neuron_step(float &u, float &syn, float zp, float in, float alpha,
                                    float beta, float jump) {
    float uu;
    if constexpr (NEURON == SNN_SYNAPTIC) {
        syn = __builtin_fmaf(alpha, syn, in);
        uu = __builtin_fmaf(beta, u, syn);
    } else {
        uu = __builtin_fmaf(beta, u, in);
    }
    uu = (zp != 0.f) ? uu + jump : uu;
    u = uu;
    return uu;
}

// Surrogate derivative of the spike at membrane u (eq. (9) with slope k):
// 1 / (1 + k |u - thr|)^2.
__device__ inline float surrogate(float u, float thr, float slope) {
    const float e = 1.f + slope * __builtin_fabsf(u - thr);
    return __builtin_amdgcn_rcpf(e * e);
}

// One reverse step of the adjoint for a Leaky or Synaptic column: with s the
// surrogate at u_t and gt = dL/dz_t,
//   lam_t = c lam_{t+1} + gt s,  c = beta (reset detached) or beta - thr s
//   (reset differentiated through the surrogate);
// the current-based neuron carries a second adjoint lami_t = alpha
// lami_{t+1} + lam_t.  Returns dL/dI_t.
template <int NEURON, bool RESET_SURR>
__device__ inline float adjoint_step(float &lam, float &lami, float gt, float s, float alpha,
                                     float beta, float thr) {
    const float carry = RESET_SURR ? beta - thr * s : beta;
    lam = __builtin_fmaf(carry, lam, gt * s);
    if constexpr (NEURON == SNN_SYNAPTIC) {
        lami = __builtin_fmaf(alpha, lami, lam);
        return lami;
    }
    return lam;
}

}  // namespace snn
