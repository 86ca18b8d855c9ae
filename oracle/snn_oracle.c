/*
 * snn_oracle.c -- plain, slow CPU oracle for spiking-layer training
 * (time-stepped forward pass, BPTT backward with a fast-sigmoid surrogate).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  It shares no code,
 * header, table or helper with the GPU library; it includes only the C
 * standard library.
 *
 * Precision (see each function):
 *   - dot products (dense and convolutional synapses, their gradients) and
 *     the adjoint recursion are evaluated in double;
 *   - the forward neuron recurrence is evaluated in fp32, the precision the
 *     method runs in (the paper's experiments use 32-bit floats by default,
 *     Sec. IV "Mixed Precision Performance"), because the fp32 membrane value
 *     decides each spike: both the oracle and the GPU take that integer
 *     decision in fp32.  The op order is: one fused multiply-add for the
 *     decay-plus-input term, then the reset subtraction (reading of eq. 4).
 *
 * Every loop reduces in a fixed order, so results do not depend on the
 * number of OpenMP threads.
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <string.h>

#define ORC_LEAKY 0
#define ORC_SYNAPTIC 1

/* ------------------------------------------------------------------------
 * Dense synapse, forward: the weighted input term "w x_t" of eqs. (4)/(5),
 * for every output neuron o and every (t,b) row m, plus a bias:
 *     I[m,o] = b[o] + sum_i W[o,i] * x[m,i]
 * x is [M, n_in] row-major (M = T*B), W is [n_out, n_in], I is [M, n_out].
 * b may be NULL.  Accumulated in double, bias first, then i ascending.
 * ---------------------------------------------------------------------- */
void orc_dense_fwd(int64_t M, int64_t n_in, int64_t n_out, const double *x,
                   const double *W, const double *b, double *I)
{
#pragma omp parallel for schedule(static)
    for (int64_t m = 0; m < M; ++m) {
        const double *xr = x + m * n_in;
        for (int64_t o = 0; o < n_out; ++o) {
            const double *wr = W + o * n_in;
            double acc = b ? b[o] : 0.0;
            for (int64_t i = 0; i < n_in; ++i)
                acc += wr[i] * xr[i];
            I[m * n_out + o] = acc;
        }
    }
}

/* ------------------------------------------------------------------------
 * Dense synapse, backward (chain rule through I = x W^T + b):
 *     dW[o,i] = sum_m dI[m,o] x[m,i]      (m ascending)
 *     db[o]   = sum_m dI[m,o]             (m ascending)
 *     dx[m,i] = sum_o dI[m,o] W[o,i]      (o ascending)
 * Any of dW, db, dx may be NULL.
 * ---------------------------------------------------------------------- */
void orc_dense_bwd(int64_t M, int64_t n_in, int64_t n_out, const double *dI,
                   const double *x, const double *W, double *dW, double *db,
                   double *dx)
{
    if (dW || db) {
#pragma omp parallel for schedule(static)
        for (int64_t o = 0; o < n_out; ++o) {
            double sb = 0.0;
            if (dW)
                for (int64_t i = 0; i < n_in; ++i)
                    dW[o * n_in + i] = 0.0;
            for (int64_t m = 0; m < M; ++m) {
                const double d = dI[m * n_out + o];
                sb += d;
                if (dW) {
                    const double *xr = x + m * n_in;
                    double *wr = dW + o * n_in;
                    for (int64_t i = 0; i < n_in; ++i)
                        wr[i] += d * xr[i];
                }
            }
            if (db)
                db[o] = sb;
        }
    }
    if (dx) {
#pragma omp parallel for schedule(static)
        for (int64_t m = 0; m < M; ++m) {
            double *xr = dx + m * n_in;
            for (int64_t i = 0; i < n_in; ++i)
                xr[i] = 0.0;
            for (int64_t o = 0; o < n_out; ++o) {
                const double d = dI[m * n_out + o];
                const double *wr = W + o * n_in;
                for (int64_t i = 0; i < n_in; ++i)
                    xr[i] += d * wr[i];
            }
        }
    }
}

/* ------------------------------------------------------------------------
 * Convolutional synapse, forward: 2-D cross-correlation with a KxK kernel,
 * stride 1, no padding, plus a bias (the "5C12" / "5C64" layers of the
 * paper's CSNN, Table I):
 *     y[n,co,oy,ox] = b[co] + sum_{c,ky,kx} w[co,c,ky,kx] x[n,c,oy+ky,ox+kx]
 * x [N,C,H,W], w [Co,C,K,K], y [N,Co,H-K+1,W-K+1].  Accumulated in double in
 * the order c, ky, kx ascending after the bias.
 * ---------------------------------------------------------------------- */
void orc_conv_fwd(int64_t N, int64_t C, int64_t H, int64_t W, int64_t Co,
                  int64_t K, const double *x, const double *w, const double *b,
                  double *y)
{
    const int64_t Ho = H - K + 1, Wo = W - K + 1;
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t n = 0; n < N; ++n)
        for (int64_t co = 0; co < Co; ++co)
            for (int64_t oy = 0; oy < Ho; ++oy)
                for (int64_t ox = 0; ox < Wo; ++ox) {
                    double acc = b ? b[co] : 0.0;
                    for (int64_t c = 0; c < C; ++c)
                        for (int64_t ky = 0; ky < K; ++ky)
                            for (int64_t kx = 0; kx < K; ++kx)
                                acc += w[((co * C + c) * K + ky) * K + kx] *
                                       x[((n * C + c) * H + oy + ky) * W + ox + kx];
                    y[((n * Co + co) * Ho + oy) * Wo + ox] = acc;
                }
}

/* ------------------------------------------------------------------------
 * Convolutional synapse, backward.  dy [N,Co,Ho,Wo] is dL/dy.
 *     dw[co,c,ky,kx] = sum_{n,oy,ox} dy[n,co,oy,ox] x[n,c,oy+ky,ox+kx]
 *     db[co]         = sum_{n,oy,ox} dy[n,co,oy,ox]
 *     dx[n,c,y,x]    = sum_{co,ky,kx} dy[n,co,y-ky,x-kx] w[co,c,ky,kx]
 *                      over the (y-ky, x-kx) that lie inside the output.
 * Any of dw, db, dx may be NULL.
 * ---------------------------------------------------------------------- */
void orc_conv_bwd(int64_t N, int64_t C, int64_t H, int64_t W, int64_t Co,
                  int64_t K, const double *dy, const double *x, const double *w,
                  double *dw, double *db, double *dx)
{
    const int64_t Ho = H - K + 1, Wo = W - K + 1;
    if (dw || db) {
#pragma omp parallel for schedule(static)
        for (int64_t co = 0; co < Co; ++co) {
            if (db) {
                double s = 0.0;
                for (int64_t n = 0; n < N; ++n)
                    for (int64_t p = 0; p < Ho * Wo; ++p)
                        s += dy[(n * Co + co) * Ho * Wo + p];
                db[co] = s;
            }
            if (dw)
                for (int64_t c = 0; c < C; ++c)
                    for (int64_t ky = 0; ky < K; ++ky)
                        for (int64_t kx = 0; kx < K; ++kx) {
                            double s = 0.0;
                            for (int64_t n = 0; n < N; ++n)
                                for (int64_t oy = 0; oy < Ho; ++oy)
                                    for (int64_t ox = 0; ox < Wo; ++ox)
                                        s += dy[((n * Co + co) * Ho + oy) * Wo + ox] *
                                             x[((n * C + c) * H + oy + ky) * W + ox + kx];
                            dw[((co * C + c) * K + ky) * K + kx] = s;
                        }
        }
    }
    if (dx) {
#pragma omp parallel for collapse(2) schedule(static)
        for (int64_t n = 0; n < N; ++n)
            for (int64_t c = 0; c < C; ++c)
                for (int64_t yy = 0; yy < H; ++yy)
                    for (int64_t xx = 0; xx < W; ++xx) {
                        double s = 0.0;
                        for (int64_t co = 0; co < Co; ++co)
                            for (int64_t ky = 0; ky < K; ++ky)
                                for (int64_t kx = 0; kx < K; ++kx) {
                                    const int64_t oy = yy - ky, ox = xx - kx;
                                    if (oy < 0 || oy >= Ho || ox < 0 || ox >= Wo)
                                        continue;
                                    s += dy[((n * Co + co) * Ho + oy) * Wo + ox] *
                                         w[((co * C + c) * K + ky) * K + kx];
                                }
                        dx[((n * C + c) * H + yy) * W + xx] = s;
                    }
    }
}

/* ------------------------------------------------------------------------
 * 2x2 max-pooling, stride 2 ("MP2" in Table I), applied to the synaptic
 * currents before the neuron.  For each window the maximum is taken over
 * (dy,dx) in row-major order (0,0),(0,1),(1,0),(1,1); a later element
 * replaces the running maximum only if strictly greater, so ties go to the
 * first maximum.  arg[] receives 2*dy+dx.  Odd trailing rows/cols are
 * dropped (floor).  x [P,H,W] (P = N*C planes) -> y [P,H/2,W/2].
 * ---------------------------------------------------------------------- */
void orc_maxpool2_fwd(int64_t P, int64_t H, int64_t W, const double *x,
                      double *y, int8_t *arg)
{
    const int64_t Hp = H / 2, Wp = W / 2;
#pragma omp parallel for schedule(static)
    for (int64_t p = 0; p < P; ++p)
        for (int64_t py = 0; py < Hp; ++py)
            for (int64_t px = 0; px < Wp; ++px) {
                double best = x[(p * H + 2 * py) * W + 2 * px];
                int a = 0;
                for (int d = 1; d < 4; ++d) {
                    const double v = x[(p * H + 2 * py + d / 2) * W + 2 * px + d % 2];
                    if (v > best) {
                        best = v;
                        a = d;
                    }
                }
                y[(p * Hp + py) * Wp + px] = best;
                arg[(p * Hp + py) * Wp + px] = (int8_t)a;
            }
}

/* Max-pool backward: the pooled gradient goes to the window element that was
 * selected in the forward pass; every other element gets zero. */
void orc_maxpool2_bwd(int64_t P, int64_t H, int64_t W, const double *dy,
                      const int8_t *arg, double *dx)
{
    const int64_t Hp = H / 2, Wp = W / 2;
#pragma omp parallel for schedule(static)
    for (int64_t p = 0; p < P; ++p) {
        for (int64_t i = 0; i < H * W; ++i)
            dx[p * H * W + i] = 0.0;
        for (int64_t py = 0; py < Hp; ++py)
            for (int64_t px = 0; px < Wp; ++px) {
                const int a = arg[(p * Hp + py) * Wp + px];
                dx[(p * H + 2 * py + a / 2) * W + 2 * px + a % 2] =
                    dy[(p * Hp + py) * Wp + px];
            }
    }
}

/* ------------------------------------------------------------------------
 * Neuron forward scan in fp32, one independent column c per (b, n), time
 * t = 0..T-1 sequential.  I and the outputs are time-major [T, C].
 *
 *   Leaky (eq. 4):      u_t = beta*u_{t-1} + I_t - z_{t-1}*thr
 *   Synaptic (eqs. 5-6): i_t = alpha*i_{t-1} + I_t
 *                        u_t = beta*u_{t-1} + i_t - z_{t-1}*thr
 *   Spike (eq. 3):       z_t = 1 if u_t > thr (strict), else 0
 *
 * Initial state u = i = 0 and z = 0 before the first step.  Each
 * decay-plus-input term is one fmaf; the reset subtracts thr afterwards.
 * u_out[t,c] holds u_t (the value compared with thr); counts[c] = sum_t z_t.
 * z_out, u_out, counts may each be NULL.
 * ---------------------------------------------------------------------- */
void orc_scan_fwd(int neuron, int64_t T, int64_t C, float alpha, float beta,
                  float thr, const float *I, uint8_t *z_out, float *u_out,
                  float *counts)
{
#pragma omp parallel for schedule(static)
    for (int64_t c = 0; c < C; ++c) {
        float u = 0.0f, syn = 0.0f;
        int zprev = 0;
        int cnt = 0;
        for (int64_t t = 0; t < T; ++t) {
            const float in = I[t * C + c];
            if (neuron == ORC_SYNAPTIC) {
                syn = fmaf(alpha, syn, in);
                u = fmaf(beta, u, syn);
            } else {
                u = fmaf(beta, u, in);
            }
            if (zprev)
                u = u - thr;
            const int z = (u > thr) ? 1 : 0;
            if (z_out)
                z_out[t * C + c] = (uint8_t)z;
            if (u_out)
                u_out[t * C + c] = u;
            cnt += z;
            zprev = z;
        }
        if (counts)
            counts[c] = (float)cnt;
    }
}

/* ------------------------------------------------------------------------
 * Smooth forward scan in double, for finite-difference checks of the
 * backward only (never part of the method).  The Heaviside output spike is
 * replaced by the smooth step S(v) = (1 + k v / (1 + k|v|)) / 2, the
 * fast sigmoid of eq. (8) rescaled to (0,1) with slope k; its derivative is
 * S'(v) = (k/2) / (1 + k|v|)^2.  The reset term uses S(u_{t-1} - thr) when
 * reset_surrogate != 0 and the hard step H(u_{t-1} - thr) otherwise (whose
 * derivative is zero almost everywhere, i.e. a detached reset).
 * z_out[t,c] = S(u_t - thr); counts[c] = sum_t z_out[t,c].
 * ---------------------------------------------------------------------- */
void orc_scan_fwd_smooth(int neuron, int64_t T, int64_t C, double alpha,
                         double beta, double thr, double slope,
                         int reset_surrogate, const double *I, double *z_out,
                         double *u_out, double *counts)
{
#pragma omp parallel for schedule(static)
    for (int64_t c = 0; c < C; ++c) {
        double u = 0.0, syn = 0.0, rprev = 0.0, cnt = 0.0;
        for (int64_t t = 0; t < T; ++t) {
            const double in = I[t * C + c];
            if (neuron == ORC_SYNAPTIC) {
                syn = alpha * syn + in;
                u = beta * u + syn;
            } else {
                u = beta * u + in;
            }
            u = u - rprev * thr;
            const double v = u - thr;
            const double z = 0.5 * (1.0 + slope * v / (1.0 + slope * fabs(v)));
            rprev = reset_surrogate ? z : (v > 0.0 ? 1.0 : 0.0);
            if (z_out)
                z_out[t * C + c] = z;
            if (u_out)
                u_out[t * C + c] = u;
            cnt += z;
        }
        if (counts)
            counts[c] = cnt;
    }
}

/* ------------------------------------------------------------------------
 * Neuron backward scan (backpropagation through time), double precision.
 * The spike's derivative is replaced by the fast-sigmoid surrogate of eq. (9)
 * with slope k:
 *     s_t = s_scale / (1 + k*|u_t - thr|)^2
 * (s_scale = 1 for the method; s_scale = k/2 turns it into S' above for the
 * smooth finite-difference check).  With g_t = dL/dz_t and lam = 0 after
 * the last step, for t = T-1 .. 0:
 *   Leaky:    lam_t = g_t s_t + (beta - r*thr*s_t) * lam_{t+1};  dI_t = lam_t
 *   Synaptic: lamu_t = g_t s_t + (beta - r*thr*s_t) * lamu_{t+1}
 *             lami_t = lamu_t + alpha * lami_{t+1};              dI_t = lami_t
 * where r = 1 if the gradient flows through the reset term (-thr*z_{t-1} in
 * eqs. 4/6), else 0.  u is the saved membrane [T, C]; g is [T, C], or [C]
 * (the same gradient for every t) when g_bcast != 0.  dI is [T, C].
 * ---------------------------------------------------------------------- */
void orc_scan_bwd(int neuron, int64_t T, int64_t C, double alpha, double beta,
                  double thr, double slope, double s_scale, int reset_surrogate,
                  const double *u, const double *g, int g_bcast, double *dI)
{
#pragma omp parallel for schedule(static)
    for (int64_t c = 0; c < C; ++c) {
        double lamu = 0.0, lami = 0.0;
        for (int64_t t = T - 1; t >= 0; --t) {
            const double v = fabs(u[t * C + c] - thr);
            const double d = 1.0 + slope * v;
            const double s = s_scale / (d * d);
            const double gt = g_bcast ? g[c] : g[t * C + c];
            const double carry = beta - (reset_surrogate ? thr * s : 0.0);
            lamu = gt * s + carry * lamu;
            if (neuron == ORC_SYNAPTIC) {
                lami = lamu + alpha * lami;
                dI[t * C + c] = lami;
            } else {
                dI[t * C + c] = lamu;
            }
        }
    }
}

/* ------------------------------------------------------------------------
 * Recurrent leaky integrate-and-fire neuron, eq. (7): the neuron's own
 * previous spike, weighted by the recurrent weight v, joins the input:
 *     u_t = beta*u_{t-1} + I_t + z_{t-1} * (v - thr)
 * One recurrent weight per neuron; column c of [T, C] (C = B*N, neuron
 * fastest) is neuron c % N.  fp32, op order of eq. (7) read left to right:
 * the decay-plus-input term is one fused multiply-add, then (v - thr), rounded
 * once to fp32, is added if the previous step spiked.  v = 0 gives eq. (4).
 * ---------------------------------------------------------------------- */
void orc_scan_fwd_rleaky(int64_t T, int64_t C, int64_t N, float beta, float thr,
                         const float *v, const float *I, uint8_t *z_out,
                         float *u_out, float *counts)
{
#pragma omp parallel for schedule(static)
    for (int64_t c = 0; c < C; ++c) {
        const float jump = v[c % N] - thr;
        float u = 0.0f;
        int zprev = 0, cnt = 0;
        for (int64_t t = 0; t < T; ++t) {
            u = fmaf(beta, u, I[t * C + c]);
            if (zprev)
                u = u + jump;
            const int z = (u > thr) ? 1 : 0;
            if (z_out)
                z_out[t * C + c] = (uint8_t)z;
            if (u_out)
                u_out[t * C + c] = u;
            cnt += z;
            zprev = z;
        }
        if (counts)
            counts[c] = (float)cnt;
    }
}

/* Smooth version in double for finite differences (not the method): the
 * spike is S(u - thr) as in orc_scan_fwd_smooth; the recurrent term uses the
 * smooth spike v * S(u_{t-1} - thr), the reset term thr * S(u_{t-1} - thr)
 * when reset_surrogate != 0, else thr * H(u_{t-1} - thr) (detached). */
void orc_scan_fwd_smooth_rleaky(int64_t T, int64_t C, int64_t N, double beta,
                                double thr, double slope, int reset_surrogate,
                                const double *v, const double *I, double *z_out,
                                double *u_out, double *counts)
{
#pragma omp parallel for schedule(static)
    for (int64_t c = 0; c < C; ++c) {
        const double vc = v[c % N];
        double u = 0.0, zprev = 0.0, rprev = 0.0, cnt = 0.0;
        for (int64_t t = 0; t < T; ++t) {
            u = beta * u + I[t * C + c] + vc * zprev - thr * rprev;
            const double d = u - thr;
            const double z = 0.5 * (1.0 + slope * d / (1.0 + slope * fabs(d)));
            zprev = z;
            rprev = reset_surrogate ? z : (d > 0.0 ? 1.0 : 0.0);
            if (z_out)
                z_out[t * C + c] = z;
            if (u_out)
                u_out[t * C + c] = u;
            cnt += z;
        }
        if (counts)
            counts[c] = cnt;
    }
}

/* BPTT through eq. (7), double.  s_t = s_scale / (1 + k|u_t - thr|)^2 as in
 * orc_scan_bwd; the spike z_t reaches u_{t+1} through (v - r*thr), so
 *     lam_t = g_t s_t + (beta + (v - r*thr) s_t) * lam_{t+1},   dI_t = lam_t,
 * and the recurrent weight collects dv_col[c] = sum_{t>=1} lam_t z_{t-1}
 * (per column; the caller sums the columns of each neuron).  z_{t-1} is the
 * method's spike H(u_{t-1} - thr), or S(u_{t-1} - thr) when smooth_z != 0 (the
 * smooth forward above). */
void orc_scan_bwd_rleaky(int64_t T, int64_t C, int64_t N, double beta, double thr,
                         double slope, double s_scale, int reset_surrogate,
                         int smooth_z, const double *v, const double *u,
                         const double *g, int g_bcast, double *dI, double *dv_col)
{
#pragma omp parallel for schedule(static)
    for (int64_t c = 0; c < C; ++c) {
        const double vc = v[c % N];
        double lam = 0.0, dv = 0.0;
        for (int64_t t = T - 1; t >= 0; --t) {
            const double e = u[t * C + c] - thr;
            const double d = 1.0 + slope * fabs(e);
            const double s = s_scale / (d * d);
            const double gt = g_bcast ? g[c] : g[t * C + c];
            lam = gt * s + (beta + (vc - (reset_surrogate ? thr : 0.0)) * s) * lam;
            dI[t * C + c] = lam;
            if (t > 0) {
                const double ep = u[(t - 1) * C + c] - thr;
                const double zp = smooth_z
                    ? 0.5 * (1.0 + slope * ep / (1.0 + slope * fabs(ep)))
                    : (ep > 0.0 ? 1.0 : 0.0);
                dv += lam * zp;
            }
        }
        if (dv_col)
            dv_col[c] = dv;
    }
}

/* ------------------------------------------------------------------------
 * Rate-coded readout loss on output spike counts (the predicted class is the
 * output neuron with the most spikes, Sec. V).  Cross-entropy with the raw
 * counts as logits, mean over the batch:
 *     L = (1/B) sum_b [ log sum_k exp(c[b,k]) - c[b,y_b] ]
 *     grad[b,k] = (softmax(c[b])_k - [k == y_b]) / B
 * The log-sum-exp subtracts the row maximum first.  Returns L.
 * ---------------------------------------------------------------------- */
double orc_loss_ce(int64_t B, int64_t K, const double *counts,
                   const int32_t *labels, double *grad)
{
    double total = 0.0;
    for (int64_t b = 0; b < B; ++b) {
        const double *c = counts + b * K;
        double mx = c[0];
        for (int64_t k = 1; k < K; ++k)
            if (c[k] > mx)
                mx = c[k];
        double se = 0.0;
        for (int64_t k = 0; k < K; ++k)
            se += exp(c[k] - mx);
        const double lse = mx + log(se);
        total += lse - c[labels[b]];
        if (grad)
            for (int64_t k = 0; k < K; ++k)
                grad[b * K + k] =
                    (exp(c[k] - mx) / se - (k == labels[b] ? 1.0 : 0.0)) / (double)B;
    }
    return total / (double)B;
}

/* Mean-squared error on spike counts against real-valued targets, mean over
 * all B*K entries:  L = (1/(B K)) sum (c - y)^2,  grad = 2 (c - y) / (B K). */
double orc_loss_mse(int64_t B, int64_t K, const double *counts,
                    const double *targets, double *grad)
{
    const int64_t n = B * K;
    double total = 0.0;
    for (int64_t j = 0; j < n; ++j) {
        const double d = counts[j] - targets[j];
        total += d * d;
        if (grad)
            grad[j] = 2.0 * d / (double)n;
    }
    return total / (double)n;
}

/* ------------------------------------------------------------------------
 * Weight update with AdamW, the optimizer the paper trains every network with
 * (Sec. IV): Adam's moment estimates with bias correction (Kingma and Ba) and
 * weight decay decoupled from the gradient (Loshchilov and Hutter), one step
 * t >= 1, in double, elementwise:
 *     theta <- theta - lr * wd * theta
 *     m     <- beta1 m + (1 - beta1) g
 *     v     <- beta2 v + (1 - beta2) g^2
 *     mhat  =  m / (1 - beta1^t),   vhat = v / (1 - beta2^t)
 *     theta <- theta - lr * mhat / (sqrt(vhat) + eps)
 * theta, m, v are updated in place.
 * ---------------------------------------------------------------------- */
void orc_adamw(int64_t n, double *theta, const double *g, double *m, double *v,
               int64_t t, double lr, double beta1, double beta2, double eps,
               double wd)
{
    const double bc1 = 1.0 - pow(beta1, (double)t);
    const double bc2 = 1.0 - pow(beta2, (double)t);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        double th = theta[i];
        th = th - lr * wd * th;
        m[i] = beta1 * m[i] + (1.0 - beta1) * g[i];
        v[i] = beta2 * v[i] + (1.0 - beta2) * g[i] * g[i];
        const double mhat = m[i] / bc1;
        const double vhat = v[i] / bc2;
        theta[i] = th - lr * mhat / (sqrt(vhat) + eps);
    }
}

/* Number of OpenMP threads a parallel region uses (for reporting). */
int orc_num_threads(void)
{
    int n = 1;
#pragma omp parallel
    {
#pragma omp single
        {
#ifdef _OPENMP
            extern int omp_get_num_threads(void);
            n = omp_get_num_threads();
#endif
        }
    }
    return n;
}
