// misc.hip -- the non-convolution kernels of the step: batch-norm
// statistics / apply / backward, ReLU, residual add, max pool, global
// average pool, channel concatenation, the plain linear layer, softmax
// cross-entropy, layout conversions,
// the replica snapshot, the block SGD update and replica averaging.
//
// Activations are NHWC, stored as float32 or bfloat16 (act.h); every kernel
// that touches them is a template over the storage type and computes in
// float32.  Batch-norm reductions are merged across workgroups either in a
// fixed order (partials and a finalize kernel) or by fp64 atomic adds into
// per-channel accumulators (bnacc.h); every other reduction runs in a fixed
// order.
#include <algorithm>
#include <mutex>

#include "act.h"
#include "bnacc.h"
#include "kernels.h"
#include "launch.h"

namespace lpp {

static inline unsigned nblocks(long n, int per) { return (unsigned)((n + per - 1) / per); }

// ------------------------------------------------------------------------
// batch-norm statistics: per row tile, per channel, the tile mean and the
// sum of squared deviations from it (two passes over the tile), written as
// partials or added to the batch sums
// ------------------------------------------------------------------------

// Row tiles of the stand-alone reductions (BN statistics and the BN
// backward's sums): about M / 128 rows, so that a tensor gives ~128
// workgroups, within [16, 512] (grid.y takes chunks of 256 channel quads).
int stats_rows(long M, int C) {
    const long gy = ((C >> 2) + 255) / 256;
    long r = (M * gy + 127) / 128;
    return (int)(r < 16 ? 16 : (r > 512 ? 512 : r));   // cap 512: +0.75% on ResNet-20 against 256 or 1024
}
int stats_tiles(long M, int C) {
    const int R = stats_rows(M, C);
    return (int)((M + R - 1) / R);
}

// Threads tile the rows x channel-quads of one row tile; quads beyond 256
// are handled in chunks.  Returns nq (quads in this chunk) and rl (row lanes).
__device__ __forceinline__ void quad_layout(int C4, int qbase, int& nq, int& rl) {
    nq = min(256, C4 - qbase);
    rl = 256 / nq;
}

template <class T>
__global__ __launch_bounds__(256) void stats_partial_k(const T* __restrict__ x, long M, int C, int R, BnSums out) {
    __shared__ f4 red[256];
    __shared__ float mean_s[1024];
    const int tid = threadIdx.x;
    const int C4 = C >> 2;
    const long r0 = (long)blockIdx.x * R;
    const long r1 = min(M, r0 + R);
    const float rows = (float)(r1 - r0);
    for (int qbase = blockIdx.y * 256; qbase < min(C4, (int)(blockIdx.y + 1) * 256); qbase += 256) {
        int nq, rl;
        quad_layout(C4, qbase, nq, rl);
        const int q = qbase + tid % nq, lr = tid / nq;
        const bool act = lr < rl;
        f4 s = f4{0.f, 0.f, 0.f, 0.f};
        if (act)
            for (long r = r0 + lr; r < r1; r += rl) s += ld4(x, r * C4 + q);
        red[tid] = s;
        __syncthreads();
        if (tid < nq) {
            f4 t = f4{0.f, 0.f, 0.f, 0.f};
            for (int l = 0; l < rl; ++l) t += red[l * nq + tid];
            for (int k = 0; k < 4; ++k) mean_s[(tid * 4 + k) & 1023] = t[k] / rows;
        }
        __syncthreads();
        f4 mu = f4{0.f, 0.f, 0.f, 0.f};
        if (act)
            for (int k = 0; k < 4; ++k) mu[k] = mean_s[((q - qbase) * 4 + k) & 1023];
        f4 v = f4{0.f, 0.f, 0.f, 0.f};
        if (act)
            for (long r = r0 + lr; r < r1; r += rl) {
                const f4 d = ld4(x, r * C4 + q) - mu;
                v += d * d;
            }
        __syncthreads();
        red[tid] = v;
        __syncthreads();
        if (tid < nq) {
            f4 t = f4{0.f, 0.f, 0.f, 0.f};
            for (int l = 0; l < rl; ++l) t += red[l * nq + tid];
            for (int k = 0; k < 4; ++k) {
                const int c = (qbase + tid) * 4 + k;
                const float mu = mean_s[(tid * 4 + k) & 1023];
                if (out.acc) {
                    const double n = (double)rows, m = (double)mu;
                    acc_add(out.acc, 0, (int)blockIdx.x, C, c, m * n);
                    acc_add(out.acc, 1, (int)blockIdx.x, C, c, (double)t[k] + n * m * m);
                } else {
                    out.p0[(long)blockIdx.x * C + c] = mu;
                    out.p1[(long)blockIdx.x * C + c] = t[k];
                }
            }
        }
        __syncthreads();
    }
}

// One workgroup per channel: thread j takes tiles j, j+256, ... and the 256
// partial sums meet in a fixed-shape LDS tree.  mean = sum n_t m_t / M,
// M2 = sum (M2_t + n_t (m_t - mean)^2).
__device__ __forceinline__ double tree_sum256(double v, double* red) {
    const int t = threadIdx.x;
    red[t] = v;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if (t < w) red[t] += red[t + w];
        __syncthreads();
    }
    const double r = red[0];
    __syncthreads();
    return r;
}

// out[c] = sum over tiles of n_t * mean_t (the column sum), fixed order
__global__ __launch_bounds__(256) void sum_from_tiles_k(const float* __restrict__ pmean, int ld, int T, int R, long M,
                                                        float* __restrict__ out) {
    __shared__ double red[256];
    const int c = blockIdx.x;
    double s = 0.0;
    for (int t = threadIdx.x; t < T; t += 256)
        s += (double)min((long)R, M - (long)t * R) * (double)pmean[(long)t * ld + c];
    s = tree_sum256(s, red);
    if (threadIdx.x == 0) out[c] = (float)s;
}

hipError_t launch_sum_from_tiles(const float* pmean, int T, int R, long M, int C, float* out, hipStream_t st) {
    launch(sum_from_tiles_k, dim3(C), dim3(256), 0, st, pmean, C, T, R, M, out);
    return hipGetLastError();
}
hipError_t launch_sum_from_tiles_ld(const float* pmean, int ld, int T, int R, long M, int C, float* out,
                                    hipStream_t st) {
    launch(sum_from_tiles_k, dim3(C), dim3(256), 0, st, pmean, ld, T, R, M, out);
    return hipGetLastError();
}

hipError_t launch_stats_partial(int dt, const void* x, long M, int C, const BnSums& out, hipStream_t st) {
    const dim3 grid(stats_tiles(M, C), ((C >> 2) + 255) / 256);
    const int R = stats_rows(M, C);
    if (dt == DT_BF16)
        launch(stats_partial_k<bf16>, grid, dim3(256), 0, st, (const bf16*)x, M, C, R, out);
    else
        launch(stats_partial_k<float>, grid, dim3(256), 0, st, (const float*)x, M, C, R, out);
    return hipGetLastError();
}

// One workgroup per channel: thread j takes tiles j, j + 256, ... and the
// partial sums meet in the fixed tree.  mean = sum n_t m_t / M,
// M2 = sum (M2_t + n_t (m_t - mean)^2).
__global__ __launch_bounds__(256) void stats_finalize_k(const float* __restrict__ pmean, const float* __restrict__ pm2,
                                                        int T, int R, long M, int C, const float* __restrict__ gamma,
                                                        const float* __restrict__ beta, float eps, float* aux) {
    __shared__ double red[256];
    const int c = blockIdx.x;
    double s = 0.0;
#pragma unroll 4
    for (int t = threadIdx.x; t < T; t += 256)
        s += (double)min((long)R, M - (long)t * R) * (double)pmean[(long)t * C + c];
    const double mu = tree_sum256(s, red) / (double)M;
    double q = 0.0;
#pragma unroll 4
    for (int t = threadIdx.x; t < T; t += 256) {
        const double d = (double)pmean[(long)t * C + c] - mu;
        q += (double)pm2[(long)t * C + c] + (double)min((long)R, M - (long)t * R) * d * d;
    }
    q = tree_sum256(q, red);
    if (threadIdx.x == 0) {
        const double r = 1.0 / sqrt(q / (double)M + (double)eps);
        const double sc = (double)gamma[c] * r;
        aux[c] = (float)mu;
        aux[C + c] = (float)r;
        aux[2 * C + c] = (float)sc;
        aux[3 * C + c] = (float)((double)beta[c] - mu * sc);
    }
}

hipError_t launch_stats_finalize(const float* pmean, const float* pm2, int T, int R, long M, int C,
                                 const float* gamma, const float* beta, float eps, float* aux, hipStream_t st) {
    launch(stats_finalize_k, dim3(C), dim3(256), 0, st, pmean, pm2, T, R, M, C, gamma, beta, eps, aux);
    return hipGetLastError();
}


// ------------------------------------------------------------------------
// batch-norm apply, fused with the residual add and the ReLU that follow it
//   y = act(x1*s1 + t1 [+ r | + x2*s2 + t2])
// ------------------------------------------------------------------------

// Each thread takes E quads (i = blockIdx.x * 256 E + u * 256 + tid) and
// issues their loads before the workgroup derives the batch-norm
// coefficients into LDS, so the two latencies overlap.
template <class T, int RES, bool RELU, int E>
__global__ __launch_bounds__(256) void bn_act_k(const T* __restrict__ x1, BnFwd b1, const T* __restrict__ r,
                                                const T* __restrict__ x2, BnFwd b2, T* __restrict__ y, long n4,
                                                int C) {
    extern __shared__ float co[];   // scale1 | shift1 | scale2 | shift2
    const long i0 = (long)blockIdx.x * 256 * E + threadIdx.x;
    f4 xa[E], xb[E];
#pragma unroll
    for (int u = 0; u < E; ++u) {
        const long i = i0 + u * 256;
        if (i < n4) {
            xa[u] = ld4(x1, i);
            if (RES == 1) xb[u] = ld4(r, i);
            if (RES == 2) xb[u] = ld4(x2, i);
        }
    }
    bn_fwd_coeffs(b1, C, co, co + C);
    if (RES == 2) bn_fwd_coeffs(b2, C, co + 2 * C, co + 3 * C);
    __syncthreads();
    const int C4 = C >> 2;
#pragma unroll
    for (int u = 0; u < E; ++u) {
        const long i = i0 + u * 256;
        if (i >= n4) continue;
        const int c = (int)((unsigned)i % (unsigned)C4) * 4;   // i < 2^31
        f4 o;
#pragma unroll
        for (int j = 0; j < 4; ++j) o[j] = __builtin_fmaf(xa[u][j], co[c + j], co[C + c + j]);
        if (RES == 1) o += xb[u];
        if (RES == 2) o += xb[u] * *(const f4*)(co + 2 * C + c) + *(const f4*)(co + 3 * C + c);
        if (RELU) {
#pragma unroll
            for (int k = 0; k < 4; ++k) o[k] = o[k] > 0.f ? o[k] : 0.f;
        }
        st4(y, i, o);
    }
}

__global__ __launch_bounds__(256) void bn_fwd_coef_k(BnFwd b, int C) {
    const int c = blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= C) return;
    const double mu = acc_read(b.acc, 0, C, c) / (double)b.M;
    double var = acc_read(b.acc, 1, C, c) / (double)b.M - mu * mu;
    var = var > 0.0 ? var : 0.0;
    const double r = 1.0 / sqrt(var + (double)b.eps);
    const double sc = (double)b.gamma[c] * r;
    b.aux[c] = (float)mu;
    b.aux[C + c] = (float)r;
    b.aux[2 * C + c] = (float)sc;
    b.aux[3 * C + c] = (float)((double)b.beta[c] - mu * sc);
}

hipError_t launch_bn_fwd_coef(const BnFwd& b, int C, hipStream_t st) {
    if (!b.acc || !b.aux) return hipErrorInvalidValue;
    launch(bn_fwd_coef_k, dim3((C + 255) / 256), dim3(256), 0, st, b, C);
    return hipGetLastError();
}

// quads per thread of the batch-norm kernels: at most about 1024 workgroups
static int bn_quads_per_thread(long n4) { return n4 > 256L * 1024 * 2 ? 4 : (n4 > 256L * 1024 ? 2 : 1); }

int bn_apply_groups(long M, int C) {
    const long n4 = M * C / 4;
    const int E = bn_quads_per_thread(n4);
    return (int)((n4 + 256L * E - 1) / (256L * E));
}

static unsigned ew_grid(long n4) {
    long b = (n4 + 255) / 256;
    return (unsigned)(b < 8192 ? (b < 1 ? 1 : b) : 8192);
}

template <class T>
static hipError_t bn_act_t(const T* x1, const BnFwd& b1, const T* r, const T* x2, const BnFwd* b2, bool relu, T* y,
                           long M, int C, hipStream_t st) {
    if (C % 4) return hipErrorInvalidValue;
    const long n4 = M * C / 4;
    const int res = r ? 1 : (x2 ? 2 : 0);
    if (res == 2 && !b2) return hipErrorInvalidValue;
    const BnFwd bb = b2 ? *b2 : BnFwd{};
    const size_t lds = sizeof(float) * 4 * C;
    const int E = bn_quads_per_thread(n4);
    const unsigned grid = (unsigned)((n4 + 256L * E - 1) / (256L * E));
#define BNACT(RS, RL, EE)                                                                                \
    launch((bn_act_k<T, RS, RL, EE>), dim3(grid), dim3(256), lds, st, x1, b1, r, x2, bb, y, n4, C)
#define BNACT_E(RS, RL) \
    do { if (E == 4) BNACT(RS, RL, 4); else if (E == 2) BNACT(RS, RL, 2); else BNACT(RS, RL, 1); } while (0)
    if (res == 0) { if (relu) BNACT_E(0, true); else BNACT_E(0, false); }
    else if (res == 1) { if (relu) BNACT_E(1, true); else BNACT_E(1, false); }
    else { if (relu) BNACT_E(2, true); else BNACT_E(2, false); }
#undef BNACT_E
#undef BNACT
    return hipGetLastError();
}

hipError_t launch_bn_act(int dt, const void* x1, const BnFwd& b1, const void* r, const void* x2, const BnFwd* b2,
                         bool relu, void* y, long M, int C, hipStream_t st) {
    if (dt == DT_BF16)
        return bn_act_t((const bf16*)x1, b1, (const bf16*)r, (const bf16*)x2, b2, relu, (bf16*)y, M, C, st);
    return bn_act_t((const float*)x1, b1, (const float*)r, (const float*)x2, b2, relu, (float*)y, M, C, st);
}

// ------------------------------------------------------------------------
// batch-norm backward, with the ReLU mask and the residual fan-out of the
// forward group folded in.  g = dy (masked by the group output > 0);
// dgamma = sum g*xhat, dbeta = sum g;
// dx = gamma*rstd*(g - mean(g) - xhat*mean(g*xhat)).
// ------------------------------------------------------------------------

// Per tile of R rows (and chunk of 256 channel quads, grid.y): threads form nq
// channel quads x rl row lanes;
// each thread's rows are loaded four at a time before use, the row lanes
// meet in a fixed-shape LDS tree, and lane 0 of each quad adds the tile's
// sums to the accumulators.
// MK: 0 no ReLU; 1 ReLU mask from the stored group output (a.mask); 2 ReLU
// decision recomputed from the BN input, relu(fma(x1, scale, shift)) > 0 with
// scale | shift at a.mask_ss (the folded forward's own expression).
template <class T, int MK, bool DUAL>
__global__ __launch_bounds__(256) void bn_bwd_reduce_k(BnBwdArgs a, int R, BnSums out) {
    const T* __restrict__ dy = (const T*)a.dy;
    const T* __restrict__ mask = (const T*)a.mask;
    const T* __restrict__ x1 = (const T*)a.x1;
    const T* __restrict__ x2 = (const T*)a.x2;
    __shared__ f4 red[3][256];
    const int tid = threadIdx.x;
    const int C = a.C, C4 = C >> 2;
    const long r0 = (long)blockIdx.x * R;
    const long r1 = min(a.M, r0 + R);
    for (int qbase = blockIdx.y * 256; qbase < min(C4, (int)(blockIdx.y + 1) * 256); qbase += 256) {
        int nq, rl;
        quad_layout(C4, qbase, nq, rl);
        const int q = qbase + tid % nq, lr = tid / nq;
        f4 s0 = f4{0.f, 0.f, 0.f, 0.f}, s1 = s0, s2 = s0;
        if (lr < rl) {
            const f4 m1 = *(const f4*)(a.mean1 + q * 4), r1v = *(const f4*)(a.rstd1 + q * 4);
            f4 msc = s0, msh = s0;
            if (MK == 2) {
                msc = *(const f4*)(a.mask_ss + q * 4);
                msh = *(const f4*)(a.mask_ss + C + q * 4);
            }
            f4 m2 = s0, r2v = s0;
            if (DUAL) {
                m2 = *(const f4*)(a.mean2 + q * 4);
                r2v = *(const f4*)(a.rstd2 + q * 4);
            }
            for (long rb = r0 + lr; rb < r1; rb += 4L * rl) {
                f4 gv[4], yv[4], xv[4], x2v[4];
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const long r = rb + (long)k * rl;
                    const long o = (r < r1 ? r : r0) * C4 + q;
                    gv[k] = ld4(dy, o);
                    if (MK == 1) yv[k] = ld4(mask, o);
                    xv[k] = ld4(x1, o);
                    if (DUAL) x2v[k] = ld4(x2, o);
                }
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    if (rb + (long)k * rl >= r1) continue;
                    f4 g = gv[k];
                    if (MK == 1) {
#pragma unroll
                        for (int j = 0; j < 4; ++j) g[j] = yv[k][j] > 0.f ? g[j] : 0.f;
                    }
                    if (MK == 2) {
#pragma unroll
                        for (int j = 0; j < 4; ++j) g[j] = __builtin_fmaf(xv[k][j], msc[j], msh[j]) > 0.f ? g[j] : 0.f;
                    }
                    s0 += g;
                    s1 += g * ((xv[k] - m1) * r1v);
                    if (DUAL) s2 += g * ((x2v[k] - m2) * r2v);
                }
            }
        }
        red[0][tid] = s0;
        red[1][tid] = s1;
        red[2][tid] = s2;
        __syncthreads();
        // fixed-shape tree over the rl row lanes (any rl): lanes [0, n - h) add lane + h
        for (int n = rl; n > 1;) {
            const int h = (n + 1) >> 1;
            if (lr < n - h) {
                const int o = (lr + h) * nq + (tid % nq);
                red[0][tid] += red[0][o];
                red[1][tid] += red[1][o];
                if (DUAL) red[2][tid] += red[2][o];
            }
            __syncthreads();
            n = h;
        }
        if (tid < nq) {
            const f4 t0 = red[0][tid], t1 = red[1][tid], t2 = red[2][tid];
            const int wg = (int)blockIdx.x;
            for (int k = 0; k < 4; ++k) {
                const int c = (qbase + tid) * 4 + k;
                if (out.acc) {
                    acc_add(out.acc, 0, wg, C, c, (double)t0[k]);
                    acc_add(out.acc, 1, wg, C, c, (double)t1[k]);
                    if (DUAL) acc_add(out.acc, 2, wg, C, c, (double)t2[k]);
                } else {
                    const long o = (long)blockIdx.x * C + c;
                    out.p0[o] = t0[k];
                    out.p1[o] = t1[k];
                    if (DUAL) out.p2[o] = t2[k];
                }
            }
        }
        __syncthreads();
    }
}

// Each thread takes E quads and issues their loads first; the prologue then
// derives per channel a = gamma*rstd, mean g, mean g*xhat (and the second
// set) from the accumulated sums, plus mean and rstd, into LDS; the first
// workgroup stores dgamma and dbeta.
template <class T, int MK, int E>
__global__ __launch_bounds__(256) void bn_bwd_apply_k(BnBwdArgs a, BnBwdCoef k, T* __restrict__ dx1, int acc1,
                                                      T* __restrict__ dx2, int acc2, T* __restrict__ dres,
                                                      int accres) {
    extern __shared__ float cf[];   // a1 | mg | mgx1 | mean1 | rstd1 | a2 | mgx2 | mean2 | rstd2
    const int C = a.C;
    const bool dual = a.x2 != nullptr;
    const long n4 = a.M * C / 4;
    const long i0 = (long)blockIdx.x * 256 * E + threadIdx.x;
    f4 gv[E], yv[E], x1v[E], x2v[E];
#pragma unroll
    for (int u = 0; u < E; ++u) {
        const long i = i0 + u * 256;
        if (i < n4) {
            gv[u] = ld4((const T*)a.dy, i);
            if (MK == 1) yv[u] = ld4((const T*)a.mask, i);
            if (dx1 || MK == 2) x1v[u] = ld4((const T*)a.x1, i);
            if (dx2) x2v[u] = ld4((const T*)a.x2, i);
        }
    }
    if (k.acc) {
        for (int c = threadIdx.x; c < C; c += blockDim.x) {
            const double t0 = acc_read(k.acc, 0, C, c), t1 = acc_read(k.acc, 1, C, c);
            cf[c] = k.gamma1[c] * a.rstd1[c];
            cf[C + c] = (float)(t0 / (double)a.M);
            cf[2 * C + c] = (float)(t1 / (double)a.M);
            cf[3 * C + c] = a.mean1[c];
            cf[4 * C + c] = a.rstd1[c];
            if (blockIdx.x == 0) {
                if (k.gg1) k.gg1[c] = (float)t1;
                if (k.gb1) k.gb1[c] = (float)t0;
            }
            if (dual) {
                const double t2 = acc_read(k.acc, 2, C, c);
                cf[5 * C + c] = k.gamma2[c] * a.rstd2[c];
                cf[6 * C + c] = (float)(t2 / (double)a.M);
                cf[7 * C + c] = a.mean2[c];
                cf[8 * C + c] = a.rstd2[c];
                if (blockIdx.x == 0) {
                    if (k.gg2) k.gg2[c] = (float)t2;
                    if (k.gb2) k.gb2[c] = (float)t0;
                }
            }
        }
    } else if (k.coef1) {
        for (int c = threadIdx.x; c < C; c += blockDim.x) {
            cf[c] = k.coef1[c];
            cf[C + c] = k.coef1[C + c];
            cf[2 * C + c] = k.coef1[2 * C + c];
            cf[3 * C + c] = a.mean1[c];
            cf[4 * C + c] = a.rstd1[c];
            if (dual && k.coef2) {
                cf[5 * C + c] = k.coef2[c];
                cf[6 * C + c] = k.coef2[2 * C + c];
                cf[7 * C + c] = a.mean2[c];
                cf[8 * C + c] = a.rstd2[c];
            }
        }
    }
    __syncthreads();
    const int C4 = C >> 2;
#pragma unroll
    for (int u = 0; u < E; ++u) {
        const long i = i0 + u * 256;
        if (i >= n4) continue;
        const int c = (int)((unsigned)i % (unsigned)C4) * 4;   // i < 2^31
        f4 g = gv[u];
        if (MK == 1) {
#pragma unroll
            for (int j = 0; j < 4; ++j) g[j] = yv[u][j] > 0.f ? g[j] : 0.f;
        }
        if (MK == 2) {
            const f4 msc = *(const f4*)(a.mask_ss + c), msh = *(const f4*)(a.mask_ss + C + c);
#pragma unroll
            for (int j = 0; j < 4; ++j) g[j] = __builtin_fmaf(x1v[u][j], msc[j], msh[j]) > 0.f ? g[j] : 0.f;
        }
        if (dx1) {
            const f4 xh = (x1v[u] - *(const f4*)(cf + 3 * C + c)) * *(const f4*)(cf + 4 * C + c);
            const f4 v = *(const f4*)(cf + c) *
                         (g - *(const f4*)(cf + C + c) - xh * *(const f4*)(cf + 2 * C + c));
            st4(dx1, i, acc1 ? ld4(dx1, i) + v : v);
        }
        if (dx2) {
            const f4 xh = (x2v[u] - *(const f4*)(cf + 7 * C + c)) * *(const f4*)(cf + 8 * C + c);
            const f4 v = *(const f4*)(cf + 5 * C + c) *
                         (g - *(const f4*)(cf + C + c) - xh * *(const f4*)(cf + 6 * C + c));
            st4(dx2, i, acc2 ? ld4(dx2, i) + v : v);
        }
        if (dres) st4(dres, i, accres ? ld4(dres, i) + g : g);
    }
}

template <class T>
static void bn_bwd_reduce_t(const BnBwdArgs& a, const BnSums& out, hipStream_t st) {
    const dim3 grid(stats_tiles(a.M, a.C), ((a.C >> 2) + 255) / 256);
    const int R = stats_rows(a.M, a.C);
    if (a.mask) {
        if (a.x2) launch((bn_bwd_reduce_k<T, 1, true>), grid, dim3(256), 0, st, a, R, out);
        else launch((bn_bwd_reduce_k<T, 1, false>), grid, dim3(256), 0, st, a, R, out);
    } else if (a.mask_ss) {
        if (a.x2) launch((bn_bwd_reduce_k<T, 2, true>), grid, dim3(256), 0, st, a, R, out);
        else launch((bn_bwd_reduce_k<T, 2, false>), grid, dim3(256), 0, st, a, R, out);
    } else {
        if (a.x2) launch((bn_bwd_reduce_k<T, 0, true>), grid, dim3(256), 0, st, a, R, out);
        else launch((bn_bwd_reduce_k<T, 0, false>), grid, dim3(256), 0, st, a, R, out);
    }
}

hipError_t launch_bn_bwd_reduce(int dt, const BnBwdArgs& a, const BnSums& out, hipStream_t st) {
    if (dt == DT_BF16) bn_bwd_reduce_t<bf16>(a, out, st);
    else bn_bwd_reduce_t<float>(a, out, st);
    return hipGetLastError();
}

__global__ __launch_bounds__(256) void bn_bwd_finalize_k(const float* __restrict__ p0, const float* __restrict__ p1,
                                                         const float* __restrict__ p2, int T, long M, int C,
                                                         const float* __restrict__ gamma1,
                                                         const float* __restrict__ rstd1, float* gg1, float* gb1,
                                                         float* coef1, const float* __restrict__ gamma2,
                                                         const float* __restrict__ rstd2, float* gg2, float* gb2,
                                                         float* coef2) {
    __shared__ double red[256];
    const int c = blockIdx.x;
    const bool dual = coef2 != nullptr;
    double s0 = 0.0, s1 = 0.0, s2 = 0.0;
#pragma unroll 4
    for (int t = threadIdx.x; t < T; t += 256) {
        s0 += (double)p0[(long)t * C + c];
        s1 += (double)p1[(long)t * C + c];
        if (dual) s2 += (double)p2[(long)t * C + c];
    }
    const double t0 = tree_sum256(s0, red);
    const double t1 = tree_sum256(s1, red);
    const double t2 = dual ? tree_sum256(s2, red) : 0.0;
    if (threadIdx.x != 0) return;
    if (gg1) gg1[c] = (float)t1;
    if (gb1) gb1[c] = (float)t0;
    coef1[c] = gamma1[c] * rstd1[c];
    coef1[C + c] = (float)(t0 / (double)M);
    coef1[2 * C + c] = (float)(t1 / (double)M);
    if (dual) {
        if (gg2) gg2[c] = (float)t2;
        if (gb2) gb2[c] = (float)t0;
        coef2[c] = gamma2[c] * rstd2[c];
        coef2[C + c] = (float)(t0 / (double)M);
        coef2[2 * C + c] = (float)(t2 / (double)M);
    }
}

__global__ __launch_bounds__(256) void bn_bwd_coef_k(BnBwdArgs a, BnBwdCoef k, float* coef1, float* coef2) {
    const int C = a.C;
    const int c = blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= C) return;
    const double t0 = acc_read(k.acc, 0, C, c), t1 = acc_read(k.acc, 1, C, c);
    coef1[c] = k.gamma1[c] * a.rstd1[c];
    coef1[C + c] = (float)(t0 / (double)a.M);
    coef1[2 * C + c] = (float)(t1 / (double)a.M);
    if (k.gg1) k.gg1[c] = (float)t1;
    if (k.gb1) k.gb1[c] = (float)t0;
    if (coef2) {
        const double t2 = acc_read(k.acc, 2, C, c);
        coef2[c] = k.gamma2[c] * a.rstd2[c];
        coef2[C + c] = (float)(t0 / (double)a.M);
        coef2[2 * C + c] = (float)(t2 / (double)a.M);
        if (k.gg2) k.gg2[c] = (float)t2;
        if (k.gb2) k.gb2[c] = (float)t0;
    }
}

hipError_t launch_bn_bwd_coef(const BnBwdArgs& a, const BnBwdCoef& k, float* coef1, float* coef2, hipStream_t st) {
    if (!k.acc || !coef1 || (coef2 && (!k.gamma2 || !a.rstd2))) return hipErrorInvalidValue;
    launch(bn_bwd_coef_k, dim3((a.C + 255) / 256), dim3(256), 0, st, a, k, coef1, coef2);
    return hipGetLastError();
}

hipError_t launch_bn_bwd_finalize(const float* p0, const float* p1, const float* p2, int T, long M, int C,
                                  const float* gamma1, const float* rstd1, float* gg1, float* gb1, float* coef1,
                                  const float* gamma2, const float* rstd2, float* gg2, float* gb2, float* coef2,
                                  hipStream_t st) {
    launch(bn_bwd_finalize_k, dim3(C), dim3(256), 0, st, p0, p1, p2, T, M, C, gamma1, rstd1, gg1, gb1,
                       coef1, gamma2, rstd2, gg2, gb2, coef2);
    return hipGetLastError();
}


template <class T>
static hipError_t bn_bwd_apply_t(const BnBwdArgs& a, const BnBwdCoef& k, T* dx1, bool acc1, T* dx2, bool acc2,
                                 T* dres, bool accres, hipStream_t st) {
    if (a.C % 4) return hipErrorInvalidValue;
    if ((dx1 || dx2) && !k.acc && !k.coef1) return hipErrorInvalidValue;
    if (dx2 && !k.acc && !k.coef2) return hipErrorInvalidValue;
    const long n4 = a.M * a.C / 4;
    const int E = bn_quads_per_thread(n4);
    // one workgroup when only dgamma and dbeta are wanted
    const unsigned grid = (dx1 || dx2 || dres) ? (unsigned)((n4 + 256L * E - 1) / (256L * E)) : 1u;
    const size_t lds = sizeof(float) * 9 * a.C;
#define BNBA(MK, EE)                                                                                         \
    launch((bn_bwd_apply_k<T, MK, EE>), dim3(grid), dim3(256), lds, st, a, k, dx1, (int)acc1, dx2, \
                       (int)acc2, dres, (int)accres)
#define BNBA_E(MK) \
    do { if (E == 4) BNBA(MK, 4); else if (E == 2) BNBA(MK, 2); else BNBA(MK, 1); } while (0)
    if (a.mask) BNBA_E(1);
    else if (a.mask_ss) BNBA_E(2);
    else BNBA_E(0);
#undef BNBA_E
#undef BNBA
    return hipGetLastError();
}

hipError_t launch_bn_bwd_apply(int dt, const BnBwdArgs& a, const BnBwdCoef& k, void* dx1, bool acc1, void* dx2,
                               bool acc2, void* dres, bool accres, hipStream_t st) {
    if (dt == DT_BF16)
        return bn_bwd_apply_t(a, k, (bf16*)dx1, acc1, (bf16*)dx2, acc2, (bf16*)dres, accres, st);
    return bn_bwd_apply_t(a, k, (float*)dx1, acc1, (float*)dx2, acc2, (float*)dres, accres, st);
}

// ------------------------------------------------------------------------
// elementwise (unfused per-layer mode)
// ------------------------------------------------------------------------

template <class T>
__global__ void relu_fwd_k(const T* __restrict__ x, T* __restrict__ y, long n4) {
    for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += (long)gridDim.x * blockDim.x) {
        f4 v = ld4(x, i);
#pragma unroll
        for (int k = 0; k < 4; ++k) v[k] = v[k] > 0.f ? v[k] : 0.f;
        st4(y, i, v);
    }
}

template <class T>
__global__ void relu_bwd_k(const T* __restrict__ dy, const T* __restrict__ x, T* __restrict__ dx, long n4, int acc) {
    for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += (long)gridDim.x * blockDim.x) {
        const f4 g = ld4(dy, i), v = ld4(x, i);
        f4 o = acc ? ld4(dx, i) : f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int k = 0; k < 4; ++k) o[k] += v[k] > 0.f ? g[k] : 0.f;
        st4(dx, i, o);
    }
}

template <class T>
__global__ void add_fwd_k(const T* __restrict__ a, const T* __restrict__ b, T* __restrict__ y, long n4) {
    for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += (long)gridDim.x * blockDim.x)
        st4(y, i, ld4(a, i) + ld4(b, i));
}

template <class T>
__global__ void copy_acc_k(const T* __restrict__ s, T* __restrict__ d, long n4, int acc) {
    for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += (long)gridDim.x * blockDim.x)
        st4(d, i, acc ? ld4(d, i) + ld4(s, i) : ld4(s, i));
}

// The gradient at a ReLU's output masked in place into the gradient at its
// input (where the stored output y is zero: the ReLU clipped), and per row
// tile of stats_rows(M, C) rows the mean over the tile of each masked
// column, pmean[tile][c] -- a conv bias gradient's partials, summed by
// sum_from_tiles.  Tiling as stats_partial_k.
template <class T>
__global__ __launch_bounds__(256) void relu_mask_colsum_k(T* __restrict__ dy, const T* __restrict__ y, long M, int C,
                                                          int R, float* __restrict__ pmean) {
    __shared__ f4 red[256];
    const int tid = threadIdx.x;
    const int C4 = C >> 2;
    const long r0 = (long)blockIdx.x * R;
    const long r1 = min(M, r0 + R);
    const float rows = (float)(r1 - r0);
    for (int qbase = blockIdx.y * 256; qbase < min(C4, (int)(blockIdx.y + 1) * 256); qbase += 256) {
        int nq, rl;
        quad_layout(C4, qbase, nq, rl);
        const int q = qbase + tid % nq, lr = tid / nq;
        f4 s = f4{0.f, 0.f, 0.f, 0.f};
        if (lr < rl)
            for (long r = r0 + lr; r < r1; r += rl) {
                f4 g = ld4(dy, r * C4 + q);
                const f4 v = ld4(y, r * C4 + q);
#pragma unroll
                for (int k = 0; k < 4; ++k) g[k] = v[k] > 0.f ? g[k] : 0.f;
                st4(dy, r * C4 + q, g);
                s += g;
            }
        red[tid] = s;
        __syncthreads();
        if (tid < nq) {
            f4 t = f4{0.f, 0.f, 0.f, 0.f};
            for (int k = 0; k < rl; ++k) t += red[k * nq + tid];
            for (int k = 0; k < 4; ++k) pmean[(long)blockIdx.x * C + (qbase + tid) * 4 + k] = t[k] / rows;
        }
        __syncthreads();
    }
}

hipError_t launch_relu_mask_colsum(int dt, void* dy, const void* y, long M, int C, float* pmean, hipStream_t st) {
    if (C % 4) return hipErrorInvalidValue;
    const dim3 grid(stats_tiles(M, C), ((C >> 2) + 255) / 256);
    const int R = stats_rows(M, C);
    if (dt == DT_BF16)
        launch(relu_mask_colsum_k<bf16>, grid, dim3(256), 0, st, (bf16*)dy, (const bf16*)y, M, C, R, pmean);
    else
        launch(relu_mask_colsum_k<float>, grid, dim3(256), 0, st, (float*)dy, (const float*)y, M, C, R, pmean);
    return hipGetLastError();
}

// Backward of a channel concatenation whose two inputs are ReLU outputs
// (each applied by its producing conv): the slices of dy, masked where the
// stored ReLU output is zero, into da and db (null: not wanted), and per row
// tile of stats_rows(M, C) rows the tile means of the masked columns,
// pmean[tile][c] over the concatenated channels c < C = ca + cb.
template <class T>
__global__ __launch_bounds__(256) void concat_relu_bwd_k(const T* __restrict__ dy, const T* __restrict__ ya,
                                                         const T* __restrict__ yb, T* __restrict__ da,
                                                         T* __restrict__ db, long M, int ca, int cb, int R,
                                                         float* __restrict__ pmean) {
    __shared__ f4 red[256];
    const int tid = threadIdx.x;
    const int C = ca + cb, C4 = C >> 2, A4 = ca >> 2, B4 = cb >> 2;
    const long r0 = (long)blockIdx.x * R;
    const long r1 = min(M, r0 + R);
    const float rows = (float)(r1 - r0);
    for (int qbase = blockIdx.y * 256; qbase < min(C4, (int)(blockIdx.y + 1) * 256); qbase += 256) {
        int nq, rl;
        quad_layout(C4, qbase, nq, rl);
        const int q = qbase + tid % nq, lr = tid / nq;
        const bool in_a = q < A4;
        const T* yv = in_a ? ya : yb;
        T* dv = in_a ? da : db;
        const int qq = in_a ? q : q - A4, cq = in_a ? A4 : B4;
        f4 s = f4{0.f, 0.f, 0.f, 0.f};
        if (lr < rl)
            for (long r = r0 + lr; r < r1; r += rl) {
                f4 g = ld4(dy, r * C4 + q);
                const f4 v = ld4(yv, r * cq + qq);
#pragma unroll
                for (int k = 0; k < 4; ++k) g[k] = v[k] > 0.f ? g[k] : 0.f;
                if (dv) st4(dv, r * cq + qq, g);
                s += g;
            }
        if (pmean) {
            red[tid] = s;
            __syncthreads();
            if (tid < nq) {
                f4 t = f4{0.f, 0.f, 0.f, 0.f};
                for (int k = 0; k < rl; ++k) t += red[k * nq + tid];
                for (int k = 0; k < 4; ++k) pmean[(long)blockIdx.x * C + (qbase + tid) * 4 + k] = t[k] / rows;
            }
            __syncthreads();
        }
    }
}

hipError_t launch_concat_relu_bwd(int dt, const void* dy, const void* ya, const void* yb, void* da, void* db, long M,
                                  int ca, int cb, float* pmean, hipStream_t st) {
    if ((ca | cb) & 3) return hipErrorInvalidValue;
    const int C = ca + cb;
    const dim3 grid(stats_tiles(M, C), ((C >> 2) + 255) / 256);
    const int R = stats_rows(M, C);
    if (dt == DT_BF16)
        launch(concat_relu_bwd_k<bf16>, grid, dim3(256), 0, st, (const bf16*)dy, (const bf16*)ya, (const bf16*)yb,
               (bf16*)da, (bf16*)db, M, ca, cb, R, pmean);
    else
        launch(concat_relu_bwd_k<float>, grid, dim3(256), 0, st, (const float*)dy, (const float*)ya,
               (const float*)yb, (float*)da, (float*)db, M, ca, cb, R, pmean);
    return hipGetLastError();
}

hipError_t launch_relu_fwd(int dt, const void* x, void* y, long n, hipStream_t st) {
    if (dt == DT_BF16)
        launch(relu_fwd_k<bf16>, dim3(ew_grid(n / 4)), dim3(256), 0, st, (const bf16*)x, (bf16*)y, n / 4);
    else
        launch(relu_fwd_k<float>, dim3(ew_grid(n / 4)), dim3(256), 0, st, (const float*)x, (float*)y,
                           n / 4);
    return hipGetLastError();
}
hipError_t launch_relu_bwd(int dt, const void* dy, const void* x, void* dx, long n, bool accumulate, hipStream_t st) {
    if (dt == DT_BF16)
        launch(relu_bwd_k<bf16>, dim3(ew_grid(n / 4)), dim3(256), 0, st, (const bf16*)dy, (const bf16*)x,
                           (bf16*)dx, n / 4, (int)accumulate);
    else
        launch(relu_bwd_k<float>, dim3(ew_grid(n / 4)), dim3(256), 0, st, (const float*)dy,
                           (const float*)x, (float*)dx, n / 4, (int)accumulate);
    return hipGetLastError();
}
hipError_t launch_add_fwd(int dt, const void* a, const void* b, void* y, long n, hipStream_t st) {
    if (dt == DT_BF16)
        launch(add_fwd_k<bf16>, dim3(ew_grid(n / 4)), dim3(256), 0, st, (const bf16*)a, (const bf16*)b,
                           (bf16*)y, n / 4);
    else
        launch(add_fwd_k<float>, dim3(ew_grid(n / 4)), dim3(256), 0, st, (const float*)a,
                           (const float*)b, (float*)y, n / 4);
    return hipGetLastError();
}
hipError_t launch_copy_acc(int dt, const void* src, void* dst, long n, bool accumulate, hipStream_t st) {
    if (dt == DT_BF16)
        launch(copy_acc_k<bf16>, dim3(ew_grid(n / 4)), dim3(256), 0, st, (const bf16*)src, (bf16*)dst,
                           n / 4, (int)accumulate);
    else
        launch(copy_acc_k<float>, dim3(ew_grid(n / 4)), dim3(256), 0, st, (const float*)src, (float*)dst,
                           n / 4, (int)accumulate);
    return hipGetLastError();
}

// ------------------------------------------------------------------------
// channel concatenation: y[r] = (a[r], b[r]) per pixel row r, ca then cb
// channels (both multiples of 4); one thread per output channel quad
// ------------------------------------------------------------------------

template <class T>
__global__ void concat_fwd_k(const T* __restrict__ a, const T* __restrict__ b, T* __restrict__ y, long rows, int aq,
                             int bq) {
    const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
    const int cq = aq + bq;
    if (i >= rows * cq) return;
    const long r = (unsigned)i / (unsigned)cq;   // i < 2^31
    const int q = (int)(i - r * cq);
    st4(y, i, q < aq ? ld4(a, r * aq + q) : ld4(b, r * bq + (q - aq)));
}

// da / db (null: not wanted) receive their slices of dy, written or added
template <class T>
__global__ void concat_bwd_k(const T* __restrict__ dy, long rows, int aq, int bq, T* __restrict__ da, int acc_a,
                             T* __restrict__ db, int acc_b) {
    const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
    const int cq = aq + bq;
    if (i >= rows * cq) return;
    const long r = (unsigned)i / (unsigned)cq;   // i < 2^31
    const int q = (int)(i - r * cq);
    const f4 g = ld4(dy, i);
    if (q < aq) {
        if (da) st4(da, r * aq + q, acc_a ? ld4(da, r * aq + q) + g : g);
    } else if (db) {
        const long j = r * bq + (q - aq);
        st4(db, j, acc_b ? ld4(db, j) + g : g);
    }
}

hipError_t launch_concat_fwd(int dt, const void* a, int ca, const void* b, int cb, void* y, long rows,
                             hipStream_t st) {
    if ((ca | cb) & 3) return hipErrorInvalidValue;
    const dim3 grid(nblocks(rows * ((ca + cb) / 4), 256));
    if (dt == DT_BF16)
        launch(concat_fwd_k<bf16>, grid, dim3(256), 0, st, (const bf16*)a, (const bf16*)b, (bf16*)y, rows, ca / 4,
               cb / 4);
    else
        launch(concat_fwd_k<float>, grid, dim3(256), 0, st, (const float*)a, (const float*)b, (float*)y, rows,
               ca / 4, cb / 4);
    return hipGetLastError();
}
hipError_t launch_concat_bwd(int dt, const void* dy, long rows, int ca, int cb, void* da, bool acc_a, void* db,
                             bool acc_b, hipStream_t st) {
    if ((ca | cb) & 3) return hipErrorInvalidValue;
    if (!da && !db) return hipSuccess;
    const dim3 grid(nblocks(rows * ((ca + cb) / 4), 256));
    if (dt == DT_BF16)
        launch(concat_bwd_k<bf16>, grid, dim3(256), 0, st, (const bf16*)dy, rows, ca / 4, cb / 4, (bf16*)da,
               (int)acc_a, (bf16*)db, (int)acc_b);
    else
        launch(concat_bwd_k<float>, grid, dim3(256), 0, st, (const float*)dy, rows, ca / 4, cb / 4, (float*)da,
               (int)acc_a, (float*)db, (int)acc_b);
    return hipGetLastError();
}

// ------------------------------------------------------------------------
// pooling
// ------------------------------------------------------------------------

// arg holds the winning tap r*k + s (first maximum in row-major scan order)
// VW consecutive channels as floats (16 bytes for VW = 16 / sizeof(T)) and back
template <int VW>
__device__ __forceinline__ void ldv(const float* p, float* v) {
    if constexpr (VW == 4) {
        const f4 t = *(const f4*)p;
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = t[e];
    } else {
        v[0] = *p;
    }
}
template <int VW>
__device__ __forceinline__ void ldv(const bf16* p, float* v) {
    if constexpr (VW == 8) {
        const uint4 t = *(const uint4*)p;
        const uint32_t w[4] = {t.x, t.y, t.z, t.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            v[2 * e] = __uint_as_float(w[e] << 16);
            v[2 * e + 1] = __uint_as_float(w[e] & 0xffff0000u);
        }
    } else {
        v[0] = from_bf16(*p);
    }
}
template <int VW>
__device__ __forceinline__ void stv(float* p, const float* v) {
    if constexpr (VW == 4) st16(p, v);
    else *p = v[0];
}
template <int VW>
__device__ __forceinline__ void stv(bf16* p, const float* v) {
    if constexpr (VW == 8) st16(p, v);
    else *p = to_bf16(v[0]);
}

// Max pool, one thread per VW consecutive channels of one output pixel
// (16-byte loads and stores; VW = 1 when C is not a multiple of the vector):
// the window's largest value, the first in (r, s) order among equals, and
// its tap r*k + s as a byte per channel.
template <class T, int VW>
__global__ __launch_bounds__(256) void maxpool_fwd_k(const T* __restrict__ x, T* __restrict__ y,
                                                     uint8_t* __restrict__ arg, int Nb, int H, int W, int C, int Ho,
                                                     int Wo, int k, int st, int pad) {
    const int CV = C / VW;
    const int idx = blockIdx.x * 256 + threadIdx.x;
    if (idx >= Nb * Ho * Wo * CV) return;
    const int cv = idx % CV;
    int t = idx / CV;
    const int q = t % Wo;
    t /= Wo;
    const int p = t % Ho, n = t / Ho;
    float m[VW];
    int am[VW];
#pragma unroll
    for (int e = 0; e < VW; ++e) {
        m[e] = -INFINITY;
        am[e] = 0;
    }
    for (int r = 0; r < k; ++r) {
        const int hi = p * st - pad + r;
        if (hi < 0 || hi >= H) continue;
        for (int s = 0; s < k; ++s) {
            const int wi = q * st - pad + s;
            if (wi < 0 || wi >= W) continue;
            float v[VW];
            ldv<VW>(x + (((long)n * H + hi) * W + wi) * C + cv * VW, v);
#pragma unroll
            for (int e = 0; e < VW; ++e)
                if (v[e] > m[e]) {
                    m[e] = v[e];
                    am[e] = r * k + s;
                }
        }
    }
    stv<VW>(y + (long)idx * VW, m);
    if constexpr (VW == 8) {
        *(uint2*)(arg + (long)idx * 8) = uint2{(uint32_t)(am[0] | am[1] << 8 | am[2] << 16 | am[3] << 24),
                                               (uint32_t)(am[4] | am[5] << 8 | am[6] << 16 | am[7] << 24)};
    } else if constexpr (VW == 4) {
        *(uint32_t*)(arg + (long)idx * 4) = (uint32_t)(am[0] | am[1] << 8 | am[2] << 16 | am[3] << 24);
    } else {
        arg[idx] = (uint8_t)am[0];
    }
}

// Gradient of the max pool, one thread per VW consecutive channels of one
// input pixel: the sum, over the windows that contain the pixel (in (p, q)
// order), of the output gradient of those whose recorded tap is this pixel.
template <class T, int VW>
__global__ __launch_bounds__(256) void maxpool_bwd_k(const T* __restrict__ dy, const uint8_t* __restrict__ arg,
                                                     T* __restrict__ dx, int Nb, int H, int W, int C, int Ho, int Wo,
                                                     int k, int st, int pad, int acc) {
    const int CV = C / VW;
    const int idx = blockIdx.x * 256 + threadIdx.x;
    if (idx >= Nb * H * W * CV) return;
    const int cv = idx % CV;
    int t = idx / CV;
    const int w = t % W;
    t /= W;
    const int h = t % H, n = t / H;
    float s[VW];
#pragma unroll
    for (int e = 0; e < VW; ++e) s[e] = 0.f;
    // windows p with p*st - pad <= h <= p*st - pad + k - 1
    const int p_lo = max(0, (h + pad - k + st) / st), p_hi = min(Ho - 1, (h + pad) / st);
    const int q_lo = max(0, (w + pad - k + st) / st), q_hi = min(Wo - 1, (w + pad) / st);
    for (int p = p_lo; p <= p_hi; ++p)
        for (int q = q_lo; q <= q_hi; ++q) {
            const int r = h - (p * st - pad), ss = w - (q * st - pad);
            if (r < 0 || r >= k || ss < 0 || ss >= k) continue;
            const int tap = r * k + ss;
            const long o = (((long)n * Ho + p) * Wo + q) * C + cv * VW;
            uint8_t a[VW];
            if constexpr (VW == 8) {
                const uint2 u = *(const uint2*)(arg + o);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    a[e] = (uint8_t)(u.x >> (8 * e));
                    a[4 + e] = (uint8_t)(u.y >> (8 * e));
                }
            } else if constexpr (VW == 4) {
                const uint32_t u = *(const uint32_t*)(arg + o);
#pragma unroll
                for (int e = 0; e < 4; ++e) a[e] = (uint8_t)(u >> (8 * e));
            } else {
                a[0] = arg[o];
            }
            bool any = false;
#pragma unroll
            for (int e = 0; e < VW; ++e) any |= a[e] == tap;
            if (!any) continue;
            float g[VW];
            ldv<VW>(dy + o, g);
#pragma unroll
            for (int e = 0; e < VW; ++e)
                if (a[e] == tap) s[e] += g[e];
        }
    if (acc) {
        float d[VW];
        ldv<VW>(dx + (long)idx * VW, d);
#pragma unroll
        for (int e = 0; e < VW; ++e) s[e] = d[e] + s[e];
    }
    stv<VW>(dx + (long)idx * VW, s);
}

template <class T>
__global__ void gap_fwd_k(const T* __restrict__ x, float* __restrict__ y, int Nb, int HW, int C) {
    const int idx = blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= Nb * C) return;
    const int n = idx / C, c = idx - n * C;
    float s = 0.f;
    for (int e = 0; e < HW; ++e) s += ld1(x, ((long)n * HW + e) * C + c);
    y[idx] = s / (float)HW;
}

template <class T>
__global__ void gap_bwd_k(const float* __restrict__ dy, T* __restrict__ dx, int Nb, int HW, int C, int acc) {
    const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= (long)Nb * HW * C) return;
    const unsigned t = (unsigned)idx / (unsigned)C;   // idx < 2^31
    const int c = (int)((unsigned)idx - t * (unsigned)C);
    const int n = (int)(t / (unsigned)HW);
    const float v = dy[n * C + c] / (float)HW;
    st1(dx, idx, acc ? ld1(dx, idx) + v : v);
}

hipError_t launch_maxpool_fwd(int dt, const void* x, void* y, uint8_t* arg, int Nb, int H, int W, int C, int Ho,
                              int Wo, int k, int stride, int pad, hipStream_t st) {
    const long total = (long)Nb * Ho * Wo * C;
    if (total >= 0x7fffffffL || (long)Nb * H * W * C >= 0x7fffffffL) return hipErrorInvalidValue;
    if (dt == DT_BF16) {
        if (C % 8 == 0)
            launch(maxpool_fwd_k<bf16, 8>, dim3(nblocks(total / 8, 256)), dim3(256), 0, st, (const bf16*)x, (bf16*)y,
                   arg, Nb, H, W, C, Ho, Wo, k, stride, pad);
        else
            launch(maxpool_fwd_k<bf16, 1>, dim3(nblocks(total, 256)), dim3(256), 0, st, (const bf16*)x, (bf16*)y,
                   arg, Nb, H, W, C, Ho, Wo, k, stride, pad);
    } else {
        if (C % 4 == 0)
            launch(maxpool_fwd_k<float, 4>, dim3(nblocks(total / 4, 256)), dim3(256), 0, st, (const float*)x,
                   (float*)y, arg, Nb, H, W, C, Ho, Wo, k, stride, pad);
        else
            launch(maxpool_fwd_k<float, 1>, dim3(nblocks(total, 256)), dim3(256), 0, st, (const float*)x,
                   (float*)y, arg, Nb, H, W, C, Ho, Wo, k, stride, pad);
    }
    return hipGetLastError();
}
hipError_t launch_maxpool_bwd(int dt, const void* dy, const uint8_t* arg, void* dx, int Nb, int H, int W, int C,
                              int Ho, int Wo, int k, int stride, int pad, bool accumulate, hipStream_t st) {
    const long total = (long)Nb * H * W * C;
    if (total >= 0x7fffffffL || (long)Nb * Ho * Wo * C >= 0x7fffffffL) return hipErrorInvalidValue;
    if (dt == DT_BF16) {
        if (C % 8 == 0)
            launch(maxpool_bwd_k<bf16, 8>, dim3(nblocks(total / 8, 256)), dim3(256), 0, st, (const bf16*)dy, arg,
                   (bf16*)dx, Nb, H, W, C, Ho, Wo, k, stride, pad, (int)accumulate);
        else
            launch(maxpool_bwd_k<bf16, 1>, dim3(nblocks(total, 256)), dim3(256), 0, st, (const bf16*)dy, arg,
                   (bf16*)dx, Nb, H, W, C, Ho, Wo, k, stride, pad, (int)accumulate);
    } else {
        if (C % 4 == 0)
            launch(maxpool_bwd_k<float, 4>, dim3(nblocks(total / 4, 256)), dim3(256), 0, st, (const float*)dy, arg,
                   (float*)dx, Nb, H, W, C, Ho, Wo, k, stride, pad, (int)accumulate);
        else
            launch(maxpool_bwd_k<float, 1>, dim3(nblocks(total, 256)), dim3(256), 0, st, (const float*)dy, arg,
                   (float*)dx, Nb, H, W, C, Ho, Wo, k, stride, pad, (int)accumulate);
    }
    return hipGetLastError();
}
hipError_t launch_gap_fwd(int dt, const void* x, float* y, int Nb, int HW, int C, hipStream_t st) {
    const dim3 grid(nblocks((long)Nb * C, 256));
    if (dt == DT_BF16)
        launch(gap_fwd_k<bf16>, grid, dim3(256), 0, st, (const bf16*)x, y, Nb, HW, C);
    else
        launch(gap_fwd_k<float>, grid, dim3(256), 0, st, (const float*)x, y, Nb, HW, C);
    return hipGetLastError();
}
hipError_t launch_gap_bwd(int dt, const float* dy, void* dx, int Nb, int HW, int C, bool accumulate, hipStream_t st) {
    const dim3 grid(nblocks((long)Nb * HW * C, 256));
    if (dt == DT_BF16)
        launch(gap_bwd_k<bf16>, grid, dim3(256), 0, st, dy, (bf16*)dx, Nb, HW, C, (int)accumulate);
    else
        launch(gap_bwd_k<float>, grid, dim3(256), 0, st, dy, (float*)dx, Nb, HW, C, (int)accumulate);
    return hipGetLastError();
}

// ------------------------------------------------------------------------
// linear head and loss
// ------------------------------------------------------------------------

// y[m][o] = b[o] + sum_i x[m][i] W[o][i], then max(y, 0) with relu.  16
// lanes per row (four rows a wave): lane l takes columns 4l + 64j as quads
// (V4: I a multiple of 4) or l + 16j, for up to 16 outputs per pass over
// the row; the 16 lane sums of an output meet in a fixed xor-shuffle tree.
// W stays in the CU cache: every row of the grid reads the same O x I.
template <bool V4>
__global__ __launch_bounds__(256) void linear_fwd_k(const float* __restrict__ x, const float* __restrict__ W,
                                                    const float* __restrict__ b, float* __restrict__ y, int Nb,
                                                    int I, int O, int relu) {
    const int l = threadIdx.x & 15;
    const long m = (long)blockIdx.x * 16 + (threadIdx.x >> 4);
    const bool live = m < Nb;
    const float* xr = x + (live ? m : 0) * I;
    for (int o0 = 0; o0 < O; o0 += 16) {
        float s[16];
#pragma unroll
        for (int j = 0; j < 16; ++j) s[j] = 0.f;
        if (V4) {
            for (int i = 4 * l; i < I; i += 64) {
                const f4 xv = *(const f4*)(xr + i);
#pragma unroll
                for (int j = 0; j < 16; ++j)
                    if (o0 + j < O) {
                        const f4 wv = *(const f4*)(W + (long)(o0 + j) * I + i);
                        s[j] += xv[0] * wv[0] + xv[1] * wv[1] + xv[2] * wv[2] + xv[3] * wv[3];
                    }
            }
        } else {
            for (int i = l; i < I; i += 16) {
                const float xv = xr[i];
#pragma unroll
                for (int j = 0; j < 16; ++j)
                    if (o0 + j < O) s[j] += xv * W[(long)(o0 + j) * I + i];
            }
        }
#pragma unroll
        for (int j = 0; j < 16; ++j)
#pragma unroll
            for (int h = 8; h > 0; h >>= 1) s[j] += __shfl_xor(s[j], h, 16);
#pragma unroll
        for (int j = 0; j < 16; ++j)
            if (live && l == j && o0 + j < O) {
                const float v = s[j] + (b ? b[o0 + j] : 0.f);
                y[m * O + o0 + j] = relu && v < 0.f ? 0.f : v;
            }
    }
}

// Weight-gradient partials of y = x W^T + b over row splits of `rows` rows:
// part_w[s][o][i] = sum over the rows m of split s of dz[m][o] x[m][i], and
// (part_b non-null) part_b[s][o] = sum over the same rows of dz[m][o] for o
// < O, zero for O <= o < O4 = ceil4(O).  One thread per column: i < I the
// weights (16 outputs per pass over the rows, dz read at row-uniform
// addresses), I <= i < I + O4 the bias.  Rows are added in order.
__global__ __launch_bounds__(256) void linear_wgrad_part_k(const float* __restrict__ dz, const float* __restrict__ x,
                                                           float* __restrict__ part_w, float* __restrict__ part_b,
                                                           int M, int I, int O, int rows) {
    const int i = blockIdx.x * 256 + threadIdx.x;
    const int sp = blockIdx.y;
    const int m0 = sp * rows, m1 = min(M, m0 + rows);
    const int O4 = (O + 3) & ~3;
    if (i < I) {
        for (int o0 = 0; o0 < O; o0 += 16) {
            float a[16];
#pragma unroll
            for (int j = 0; j < 16; ++j) a[j] = 0.f;
            for (int m = m0; m < m1; ++m) {
                const float xv = x[(long)m * I + i];
#pragma unroll
                for (int j = 0; j < 16; ++j)
                    if (o0 + j < O) a[j] += dz[(long)m * O + o0 + j] * xv;
            }
#pragma unroll
            for (int j = 0; j < 16; ++j)
                if (o0 + j < O) part_w[((long)sp * O + o0 + j) * I + i] = a[j];
        }
    } else if (part_b && i < I + O4) {
        const int o = i - I;
        float a = 0.f;
        if (o < O)
            for (int m = m0; m < m1; ++m) a += dz[(long)m * O + o];
        part_b[(long)sp * O4 + o] = a;
    }
}

// gW[o][i] = sum_n dz[n][o] x[n][i]; gb[o] = sum_n dz[n][o]
__global__ void linear_bwd_w_k(const float* __restrict__ dz, const float* __restrict__ x, float* __restrict__ gW,
                               float* __restrict__ gb, int Nb, int I, int O) {
    const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx < (long)O * I) {
        const int o = (int)(idx / I), i = (int)(idx - (long)o * I);
        float s = 0.f;
        for (int n = 0; n < Nb; ++n) s += dz[(long)n * O + o] * x[(long)n * I + i];
        gW[idx] = s;
    } else if (gb && idx < (long)O * I + O) {
        const int o = (int)(idx - (long)O * I);
        float s = 0.f;
        for (int n = 0; n < Nb; ++n) s += dz[(long)n * O + o];
        gb[o] = s;
    }
}

__global__ void linear_bwd_x_k(const float* __restrict__ dz, const float* __restrict__ W, float* __restrict__ dx,
                               int Nb, int I, int O, int acc) {
    const int idx = blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= Nb * I) return;
    const int n = idx / I, i = idx - n * I;
    float s = 0.f;
    for (int o = 0; o < O; ++o) s += dz[(long)n * O + o] * W[(long)o * I + i];
    dx[idx] = acc ? dx[idx] + s : s;
}

// One thread per sample (classes looped); per-sample losses go to
// loss_per; loss_mean_k sums them in sample order.
__global__ void softmax_ce_k(const float* __restrict__ z, const StepArgs* __restrict__ args,
                             float* __restrict__ dz, float* __restrict__ loss_per, int Nb, int Cls) {
    const int n = blockIdx.x * blockDim.x + threadIdx.x;
    if (n >= Nb) return;
    const float* zr = z + (long)n * Cls;
    float mx = -INFINITY;
    for (int j = 0; j < Cls; ++j) mx = fmaxf(mx, zr[j]);
    float se = 0.f;
    for (int j = 0; j < Cls; ++j) se += expf(zr[j] - mx);
    const float lse = mx + logf(se);
    const int y = args->labels[n];
    for (int j = 0; j < Cls; ++j) dz[(long)n * Cls + j] = (expf(zr[j] - lse) - (j == y ? 1.f : 0.f)) / (float)Nb;
    loss_per[n] = lse - zr[y];
}

__global__ void loss_mean_k(const float* __restrict__ loss_per, int Nb, float* __restrict__ loss) {
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    float s = 0.f;
    for (int n = 0; n < Nb; ++n) s += loss_per[n];
    loss[0] = s / (float)Nb;
}

hipError_t launch_linear_fwd(const float* x, const float* W, const float* b, float* y, int Nb, int I, int O,
                             hipStream_t st, bool relu) {
    const dim3 grid((unsigned)((Nb + 15) / 16));
    if (I % 4 == 0 && ((uintptr_t)x & 15) == 0 && ((uintptr_t)W & 15) == 0)
        launch(linear_fwd_k<true>, grid, dim3(256), 0, st, x, W, b, y, Nb, I, O, (int)relu);
    else
        launch(linear_fwd_k<false>, grid, dim3(256), 0, st, x, W, b, y, Nb, I, O, (int)relu);
    return hipGetLastError();
}
int linear_wgrad_rows(long M) {
    long r = (M + kLinWgMaxSplits - 1) / kLinWgMaxSplits;
    return (int)(r < 32 ? 32 : r);
}
int linear_wgrad_splits(long M) {
    const long r = linear_wgrad_rows(M);
    return (int)((M + r - 1) / r);
}
hipError_t launch_linear_wgrad_part(const float* dz, const float* x, float* part_w, float* part_b, int M, int I,
                                    int O, hipStream_t st) {
    if (M < 1 || I < 1 || O < 1) return hipErrorInvalidValue;
    const int O4 = (O + 3) & ~3;
    const dim3 grid((unsigned)((I + (part_b ? O4 : 0) + 255) / 256), (unsigned)linear_wgrad_splits(M));
    launch(linear_wgrad_part_k, grid, dim3(256), 0, st, dz, x, part_w, part_b, M, I, O, linear_wgrad_rows(M));
    return hipGetLastError();
}
hipError_t launch_linear_bwd_w(const float* dz, const float* x, float* gW, float* gb, int Nb, int I, int O,
                               hipStream_t st) {
    launch(linear_bwd_w_k, dim3(nblocks((long)O * I + O, 256)), dim3(256), 0, st, dz, x, gW, gb, Nb, I,
                       O);
    return hipGetLastError();
}
hipError_t launch_linear_bwd_x(const float* dz, const float* W, float* dx, int Nb, int I, int O, bool accumulate,
                               hipStream_t st) {
    launch(linear_bwd_x_k, dim3(nblocks((long)Nb * I, 256)), dim3(256), 0, st, dz, W, dx, Nb, I, O,
                       (int)accumulate);
    return hipGetLastError();
}
hipError_t launch_softmax_ce(const float* z, const StepArgs* args, float* dz, float* loss, int Nb, int Cls,
                             hipStream_t st) {
    // per-sample losses live just after the loss scalar (caller sizes loss to 1 + Nb floats)
    launch(softmax_ce_k, dim3(nblocks(Nb, 64)), dim3(64), 0, st, z, args, dz, loss + 1, Nb, Cls);
    launch(loss_mean_k, dim3(1), dim3(64), 0, st, loss + 1, Nb, loss);
    return hipGetLastError();
}

// ------------------------------------------------------------------------
// layouts
// ------------------------------------------------------------------------

// One thread per pixel: the C channel values from the C planes (consecutive
// threads read consecutive pixels of a plane), written as 16-byte vectors of
// the padded channel row (channels C..Cp-1 zero).  The first n_zero doubles
// of `zero` (the step's fp64 accumulators) are cleared on the way.
template <class T>
__global__ __launch_bounds__(256) void nchw_to_nhwc_k(const StepArgs* __restrict__ args, T* __restrict__ d, int Nb,
                                                      int C, int H, int W, int Cp, double* __restrict__ zero,
                                                      long n_zero) {
    constexpr int VW = 16 / (int)sizeof(T);
    const float* __restrict__ s = args->images;
    const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
    for (long z = idx; z < n_zero; z += (long)gridDim.x * blockDim.x) zero[z] = 0.0;
    const long hw = (long)H * W;
    if (idx >= (long)Nb * hw) return;
    const long n = idx / hw;
    const float* __restrict__ sp = s + n * C * hw + (idx - n * hw);
    for (int c0 = 0; c0 < Cp; c0 += VW) {
        float vals[VW];
#pragma unroll
        for (int u = 0; u < VW; ++u) vals[u] = c0 + u < C ? sp[(long)(c0 + u) * hw] : 0.f;
        st16(d + idx * Cp + c0, vals);
    }
}

template <class T>
__global__ void nhwc_to_nchw_k(const T* __restrict__ s, float* __restrict__ d, int Nb, int C, int H, int W, int Cp) {
    const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
    const long total = (long)Nb * C * H * W;
    if (idx >= total) return;
    const int w = (int)(idx % W);
    long t = idx / W;
    const int h = (int)(t % H);
    t /= H;
    const int c = (int)(t % C);
    const int n = (int)(t / C);
    d[idx] = ld1(s, (((long)n * H + h) * W + w) * Cp + c);
}

hipError_t launch_nchw_to_nhwc(int dt, const StepArgs* args, void* dst, int Nb, int C, int H, int W, int Cp,
                               double* zero, long n_zero, hipStream_t st) {
    if (Cp % (dt == DT_BF16 ? 8 : 4) || C > Cp) return hipErrorInvalidValue;
    const dim3 grid(nblocks((long)Nb * H * W, 256));
    if (dt == DT_BF16)
        launch(nchw_to_nhwc_k<bf16>, grid, dim3(256), 0, st, args, (bf16*)dst, Nb, C, H, W, Cp, zero,
                           n_zero);
    else
        launch(nchw_to_nhwc_k<float>, grid, dim3(256), 0, st, args, (float*)dst, Nb, C, H, W, Cp, zero,
                           n_zero);
    return hipGetLastError();
}
hipError_t launch_nhwc_to_nchw(int dt, const void* src, float* dst, int Nb, int C, int H, int W, int Cp,
                               hipStream_t st) {
    const dim3 grid(nblocks((long)Nb * H * W * C, 256));
    if (dt == DT_BF16)
        launch(nhwc_to_nchw_k<bf16>, grid, dim3(256), 0, st, (const bf16*)src, dst, Nb, C, H, W, Cp);
    else
        launch(nhwc_to_nchw_k<float>, grid, dim3(256), 0, st, (const float*)src, dst, Nb, C, H, W, Cp);
    return hipGetLastError();
}

__global__ void set_step_args_k(StepArgs* dst, const float* images, const int* labels, float lr, long trace_slot) {
    if (threadIdx.x == 0 && blockIdx.x == 0) {
        dst->images = images;
        dst->labels = labels;
        dst->lr = lr;
        dst->trace_slot = trace_slot;
    }
}

hipError_t launch_set_step_args(StepArgs* dst, const float* images, const int* labels, float lr, long trace_slot,
                                hipStream_t st) {
    launch(set_step_args_k, dim3(1), dim3(64), 0, st, dst, images, labels, lr, trace_slot);
    return hipGetLastError();
}

// slot from the step arguments (args non-null) or from the argument
__global__ void timestamp_k(unsigned long long* log, const StepArgs* args, long slot, int k) {
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    const long s = args ? args->trace_slot : slot;
    if (s >= 0) log[s * 4 + k] = wall_clock64();
}

hipError_t launch_timestamp(unsigned long long* log, const StepArgs* args, long slot, int k, hipStream_t st) {
    launch(timestamp_k, dim3(1), dim3(64), 0, st, log, args, slot, k);
    return hipGetLastError();
}

// ------------------------------------------------------------------------
// snapshot, block update, averaging
// ------------------------------------------------------------------------

// floor(n / d) for n * d < 2^32: n itself for d == 1, else the high word of
// n * m with m = ceil(2^32 / d) (snap_magic, once per workgroup).  With
// n = q d + r the product n m / 2^32 exceeds q + r/d by less than n / 2^32,
// which keeps it below q + 1 while n d < 2^32.
__device__ __forceinline__ unsigned snap_magic(unsigned d) { return d <= 1 ? 0u : 0xffffffffu / d + 1u; }
__device__ __forceinline__ unsigned snap_div(unsigned n, unsigned d, unsigned m) {
    return d <= 1 ? n : __umulhi(n, m);
}

constexpr int kSnapThreads = 256;

// One workgroup per table tile.  The entry is found by a binary search over
// the entries' first workgroups (uniform, once per workgroup).  Copy entries
// move up to kSnapCopy floats in 16-byte quads (partial quads at the ends
// element by element).  A conv tile loads kt output channels' rows of ct
// input channels x R*S taps (contiguous runs of the canonical tensor, 16-byte
// loads where the runs are aligned, all issued before any LDS store) into LDS
// rows of odd pitch, then writes the W_f rows (one tap of one output channel:
// ct input channels) and the W_d rows (one tap of one input channel: kt
// output channels) as 16-byte vectors.
template <class T>
__global__ __launch_bounds__(kSnapThreads) void snapshot_k(const float* __restrict__ x, float* __restrict__ v,
                                                           const SnapEntry* __restrict__ tab, int n_ent,
                                                           T* __restrict__ wb) {
    constexpr int VW = 16 / (int)sizeof(T);
    __shared__ float sm[kSnapLds + 64];
    const long b = blockIdx.x;
    int lo = 0, hi = n_ent - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (tab[mid].tile0 <= b) lo = mid;
        else hi = mid - 1;
    }
    const SnapEntry& E = tab[lo];
    const int tid = threadIdx.x;
    const long t = b - E.tile0;
    if (E.kind == 0) {
        // chunk t of the quad-aligned run from (src & ~3)
        const long base = (E.src & ~3L) + t * kSnapCopy;
        const long e0 = base > E.src ? base : E.src;
        const long e1 = base + kSnapCopy < E.src + E.n ? base + kSnapCopy : E.src + E.n;
        constexpr int U = kSnapCopy / 4 / kSnapThreads;
        f4 buf[U];
#pragma unroll
        for (int j = 0; j < U; ++j) {
            const long a = base + 4L * (tid + j * kSnapThreads);
            if (a >= e0 && a + 4 <= e1) buf[j] = *(const f4*)(x + a);
        }
#pragma unroll
        for (int j = 0; j < U; ++j) {
            const long a = base + 4L * (tid + j * kSnapThreads);
            if (a >= e1 || a + 4 <= e0) continue;
            if (a >= e0 && a + 4 <= e1) {
                *(f4*)(v + a) = buf[j];
            } else {
                for (long e = a; e < a + 4; ++e)
                    if (e >= e0 && e < e1) v[e] = x[e];
            }
        }
        return;
    }
    const int RS = E.RS, cout = E.cout, cin = E.cin, cin_p = E.cin_p;
    const int kti = (int)(t % E.nkt), cti = (int)(t / E.nkt);
    const int k0 = kti * E.kt, c0 = cti * E.ct;
    const int ktn = min(E.kt, cout - k0);          // output channels of the tile
    const int ctn = min(E.ct, cin - c0);           // input channels loaded
    const int ctf = c0 + E.ct >= cin ? cin_p - c0 : E.ct;   // W_f channels written (the last tile pads to cin_p)
    const int rowlen = ctn * RS;
    const int pitch = rowlen | 1;
    const long rstride = (long)cin * RS;
    const float* __restrict__ src = x + E.src + (long)k0 * rstride + (long)c0 * RS;
    if (((E.src + (long)k0 * rstride + (long)c0 * RS) & 3) == 0 && (rstride & 3) == 0 && (rowlen & 3) == 0) {
        const unsigned nq = (unsigned)rowlen >> 2, mq = snap_magic(nq);
        const unsigned tot = (unsigned)ktn * nq;
        constexpr int U = kSnapLds / 4 / kSnapThreads;
        f4 buf[U];
#pragma unroll
        for (int j = 0; j < U; ++j) {
            const unsigned i = tid + j * kSnapThreads;
            if (i < tot) {
                const unsigned kk = snap_div(i, nq, mq), qq = i - kk * nq;
                buf[j] = *(const f4*)(src + (long)kk * rstride + 4 * qq);
            }
        }
#pragma unroll
        for (int j = 0; j < U; ++j) {
            const unsigned i = tid + j * kSnapThreads;
            if (i < tot) {
                const unsigned kk = snap_div(i, nq, mq), qq = i - kk * nq;
                float* d = sm + kk * pitch + 4 * qq;
                d[0] = buf[j][0];
                d[1] = buf[j][1];
                d[2] = buf[j][2];
                d[3] = buf[j][3];
            }
        }
    } else {
        const unsigned mr = snap_magic(rowlen);
        const unsigned tot = (unsigned)ktn * rowlen;
        for (unsigned i = tid; i < tot; i += kSnapThreads) {
            const unsigned kk = snap_div(i, rowlen, mr), j = i - kk * rowlen;
            sm[kk * pitch + j] = src[(long)kk * rstride + j];
        }
    }
    __syncthreads();
    const unsigned mrs = snap_magic(RS);
    {   // W_f rows: (output channel kk, tap rs) -> ctf input channels, VW per lane
        const int nch = ctf / VW;
        int lg = 0;
        while ((1 << lg) < nch) ++lg;
        const int chunk = tid & ((1 << lg) - 1);
        const int rows = ktn * RS;
        if (chunk < nch)
            for (int r = tid >> lg; r < rows; r += kSnapThreads >> lg) {
                const int kk = (int)snap_div(r, RS, mrs), rs = r - kk * RS;
                float vals[VW];
#pragma unroll
                for (int u = 0; u < VW; ++u) {
                    const int cc = chunk * VW + u;
                    vals[u] = cc < ctn ? sm[kk * pitch + cc * RS + rs] : 0.f;
                }
                st16(wb + E.dst_f + ((long)(k0 + kk) * RS + rs) * cin_p + c0 + chunk * VW, vals);
            }
    }
    {   // W_d rows: (input channel cc, tap rs) -> ktn output channels, VW per lane
        const int nch = ktn / VW;
        int lg = 0;
        while ((1 << lg) < nch) ++lg;
        const int chunk = tid & ((1 << lg) - 1);
        const int rows = ctn * RS;
        if (chunk < nch)
            for (int r = tid >> lg; r < rows; r += kSnapThreads >> lg) {
                const int cc = (int)snap_div(r, RS, mrs), rs = r - cc * RS;
                float vals[VW];
#pragma unroll
                for (int u = 0; u < VW; ++u) vals[u] = sm[(chunk * VW + u) * pitch + cc * RS + rs];
                st16(wb + E.dst_d + ((long)(c0 + cc) * RS + rs) * cout + k0 + chunk * VW, vals);
            }
    }
}

long snapshot_table(const SnapConvDesc* convs, int n_convs, long d, int dt, SnapEntry* out, int max_out,
                    int* n_out, double* bytes) {
    const int VW = dt == DT_BF16 ? 8 : 4;
    const double eb = dt == DT_BF16 ? 2.0 : 4.0;
    int n = 0;
    long tiles = 0, pos = 0;
    double by = 0.0;
    if (n_convs < 0 || d < 0 || max_out < 2 * n_convs + 1) return -1;
    auto add_copy = [&](long a, long e) {
        if (e <= a) return;
        SnapEntry& c = out[n++];
        c = SnapEntry{};
        c.kind = 0;
        c.src = a;
        c.n = e - a;
        c.tile0 = tiles;
        tiles += (e - (a & ~3L) + kSnapCopy - 1) / kSnapCopy;
        by += 8.0 * (double)(e - a);
    };
    auto rup = [](int a, int m) { return (a + m - 1) / m * m; };
    for (int i = 0; i < n_convs; ++i) {
        const SnapConvDesc& c = convs[i];
        const int RS = c.R * c.S;
        if (c.src < pos || c.cout % VW || c.cin_p % VW || c.cin > c.cin_p || RS < 1 || c.cout < 1 || c.cin < 1 ||
            c.src + (long)c.cout * c.cin * RS > d)
            return -1;
        add_copy(pos, c.src);
        int kt = RS == 1 ? 64 : 32, ct = RS == 1 ? 128 : 32;
        kt = std::min(kt, rup(c.cout, VW));
        ct = std::min(ct, rup(c.cin, VW));
        while ((long)kt * ct * RS > kSnapLds && ct > VW) ct = std::max(VW, ct / 2 / VW * VW);
        while ((long)kt * ct * RS > kSnapLds && kt > VW) kt = std::max(VW, kt / 2 / VW * VW);
        if ((long)kt * ct * RS > kSnapLds) return -1;
        SnapEntry& e = out[n++];
        e = SnapEntry{};
        e.kind = 1;
        e.src = c.src;
        e.dst_f = c.dst_f;
        e.dst_d = c.dst_d;
        e.tile0 = tiles;
        e.cout = c.cout;
        e.cin = c.cin;
        e.cin_p = c.cin_p;
        e.RS = RS;
        e.kt = kt;
        e.ct = ct;
        e.nkt = (c.cout + kt - 1) / kt;
        tiles += (long)e.nkt * ((c.cin + ct - 1) / ct);
        const long nw = (long)c.cout * c.cin * RS;
        by += (4.0 + 2.0 * eb) * (double)nw;
        pos = c.src + nw;
    }
    add_copy(pos, d);
    if (bytes) *bytes = by;
    *n_out = n;
    return tiles;
}

// The snapshot's work table for callers that cannot allocate device memory:
// a file-scope array on every device the library runs on (held until the
// process ends).  Host code reaches it only through the address
// hipGetSymbolAddress returns for the current device (snap_scratch_ptr);
// the array's name itself is a host-side stand-in.
static __device__ __align__(256) SnapEntry scratch[kSnapScratchEntries];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
SnapEntry* g_scratch_ptr[kMaxDevices] = {};

// scratch's address on the current device, looked up once per device
hipError_t snap_scratch_ptr(SnapEntry** out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> g(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        g_scratch_ptr[dev] = (SnapEntry*)p;
    }
    *out = g_scratch_ptr[dev];
    return hipSuccess;
}
}  // namespace

hipError_t snapshot_noalloc(int dt, const SnapConvDesc* convs, int n_convs, long d, const float* x, float* v,
                            void* wbase, hipStream_t st, int* bad_list) {
    *bad_list = 0;
    SnapEntry tab[kSnapScratchEntries];
    int n_ent = 0;
    if (n_convs > kSnapNoallocConvs) {
        *bad_list = 1;
        return hipSuccess;
    }
    const long tiles = snapshot_table(convs, n_convs, d, dt, tab, kSnapScratchEntries, &n_ent, nullptr);
    if (tiles < 0) {
        *bad_list = 1;
        return hipSuccess;
    }
    if (n_ent == 0 || tiles == 0) return hipSuccess;
    SnapEntry* dev_tab = nullptr;
    hipError_t e = snap_scratch_ptr(&dev_tab);
    if (e != hipSuccess) return e;
    e = hipMemcpyAsync(dev_tab, tab, sizeof(SnapEntry) * n_ent, hipMemcpyHostToDevice, st);
    if (e != hipSuccess) return e;
    e = launch_snapshot(dt, x, v, dev_tab, n_ent, tiles, wbase, st);
    if (e != hipSuccess) return e;
    // the host table above lives on this stack frame: return only once the
    // copy (and the kernel after it) has run
    return hipStreamSynchronize(st);
}

hipError_t launch_snapshot(int dt, const float* x, float* v, const SnapEntry* tab_dev, int n_ent, long n_tiles,
                           void* wbase, hipStream_t st) {
    if (n_ent <= 0 || n_tiles <= 0) return hipSuccess;
    if (dt == DT_BF16)
        launch(snapshot_k<bf16>, dim3((unsigned)n_tiles), dim3(kSnapThreads), 0, st, x, v, tab_dev, n_ent,
               (bf16*)wbase);
    else
        launch(snapshot_k<float>, dim3((unsigned)n_tiles), dim3(kSnapThreads), 0, st, x, v, tab_dev, n_ent,
               (float*)wbase);
    return hipGetLastError();
}

// The index space is cut into aligned quads [4q, 4q+4) from the aligned start
// below lo.  Each thread takes kUpdQuads quads per pass (strided by the
// workgroup size) and issues all their loads before any arithmetic, so
// several 16-byte loads per thread are in flight; whole quads use
// nontemporal 16-byte accesses (streamed once, no reuse within the kernel),
// the quads cut by lo or hi fall back to scalar accesses.
constexpr int kUpdQuads = 4;

__device__ __forceinline__ void update_quad(f4& xv, f4& mv, const f4 gv, bool mom, float lr, float mu, float wd) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const float dir = gv[k] + wd * xv[k];
        if (mom) {
            mv[k] = mu * mv[k] + dir;
            xv[k] -= lr * mv[k];
        } else {
            xv[k] -= lr * dir;
        }
    }
}

__global__ __launch_bounds__(256) void sgd_update_k(float* __restrict__ x, float* __restrict__ m,
                                                    const float* __restrict__ g, long lo, long hi,
                                                    const StepArgs* __restrict__ args, float lr_value, float mu,
                                                    float wd) {
    const float lr = args ? args->lr : lr_value;
    const long base = lo & ~3L;
    const long nq = (hi - base + 3) / 4;
    const bool mom = m != nullptr;
    const long stride = (long)gridDim.x * blockDim.x * kUpdQuads;
    for (long q0 = (long)blockIdx.x * blockDim.x * kUpdQuads + threadIdx.x; q0 < nq; q0 += stride) {
        f4 xv[kUpdQuads], mv[kUpdQuads], gv[kUpdQuads];
        bool whole[kUpdQuads];
#pragma unroll
        for (int u = 0; u < kUpdQuads; ++u) {
            const long q = q0 + (long)u * blockDim.x;
            const long e0 = base + 4 * q;
            whole[u] = q < nq && e0 >= lo && e0 + 4 <= hi;
            if (whole[u]) {
                xv[u] = __builtin_nontemporal_load((const f4*)(x + e0));
                gv[u] = __builtin_nontemporal_load((const f4*)(g + e0));
                if (mom) mv[u] = __builtin_nontemporal_load((const f4*)(m + e0));
            }
        }
#pragma unroll
        for (int u = 0; u < kUpdQuads; ++u) {
            const long q = q0 + (long)u * blockDim.x;
            if (q >= nq) continue;
            const long e0 = base + 4 * q;
            if (whole[u]) {
                update_quad(xv[u], mv[u], gv[u], mom, lr, mu, wd);
                if (mom) __builtin_nontemporal_store(mv[u], (f4*)(m + e0));
                __builtin_nontemporal_store(xv[u], (f4*)(x + e0));
            } else {
                for (long e = e0; e < e0 + 4; ++e) {
                    if (e < lo || e >= hi) continue;
                    float dir = g[e] + wd * x[e];
                    if (mom) {
                        m[e] = mu * m[e] + dir;
                        dir = m[e];
                    }
                    x[e] -= lr * dir;
                }
            }
        }
    }
}

hipError_t launch_sgd_update(float* x, float* m, const float* g, long lo, long hi, const StepArgs* args, float lr,
                             float mu, float wd, hipStream_t st) {
    if (hi <= lo) return hipSuccess;
    const long nq = (hi - (lo & ~3L) + 3) / 4;
    long b = (nq + 256L * kUpdQuads - 1) / (256L * kUpdQuads);
    if (b > (1L << 20)) b = 1L << 20;   // one pass up to 4G parameters (5.84 against 5.73 TB/s on 1 GiB arrays)
    launch(sgd_update_k, dim3((unsigned)b), dim3(256), 0, st, x, m, g, lo, hi, args, lr, mu, wd);
    return hipGetLastError();
}

// v_k = x_k[e]; vbar = (sum_k v_k) / n; x_k[e] = x_k[e] (re-read) + (vbar - v_k).
// U quads per thread per pass (1 in use), 512-thread workgroups.  The re-read
// of x_k is a device-scope (sc1) 16-byte buffer load: it cannot be merged
// with the first read and does not hit the compute unit's own cache, so a
// block update that another stream's kernel has written back between the two
// reads is kept (Alg. 1's averager adds vbar - v_k to x_k in place).  The
// window is not closed: an update landing after the re-read, or still held in
// another XCD's cache, is overwritten -- a lost update, which the lock-free
// updaters of the method permit.  The result is stored nontemporally (x_k is
// streamed once).
constexpr int kAvgThreads = 512;
// one quad per thread over the whole array up to 512M quads (measured on
// 1 GiB replicas: 5.71 TB/s against 5.53 with a two-pass grid-stride loop
// over 65536 workgroups)
constexpr long kAvgMaxBlocks = 1L << 20;

__device__ __forceinline__ float reread(const float* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// 16 bytes at base + byte_off (base uniform across the wave) with cache
// policy sc1: a device-scope load that bypasses the compute unit's cache
__device__ __forceinline__ f4 reread4(const float* base, unsigned byte_off) {
    const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc((void*)base, (short)0, 0x7fffffff, 0x00020000);
    return __builtin_bit_cast(f4, __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, 0, 16));
}

template <int NR, int U>
__global__ __launch_bounds__(kAvgThreads) void average_k(RepPtrs reps, int n_rep, long n) {
    const long nq = n / 4;
    const float inv_div = (float)n_rep;
    const long stride = (long)gridDim.x * blockDim.x;
    for (long q0 = (long)blockIdx.x * blockDim.x + threadIdx.x; q0 < nq; q0 += stride * U) {
        f4 v[U][NR];
        f4 vbar[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const long q = q0 + u * stride;
#pragma unroll
            for (int k = 0; k < NR; ++k)
                if (k < n_rep && q < nq) v[u][k] = *(const f4*)(reps.p[k] + 4 * q);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            f4 s = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int k = 0; k < NR; ++k)
                if (k < n_rep) s += v[u][k];
            vbar[u] = s / inv_div;
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const long q = q0 + u * stride;
#pragma unroll
            for (int k = 0; k < NR; ++k)
                if (k < n_rep && q < nq) {
                    const long qb = q - threadIdx.x;        // the workgroup's first quad (uniform)
                    const f4 cur = reread4(reps.p[k] + 4 * qb, 16u * threadIdx.x);
                    __builtin_nontemporal_store(cur + (vbar[u] - v[u][k]), (f4*)(reps.p[k] + 4 * q));   // streamed out
                }
        }
    }
    // scalar tail
    const long t0 = nq * 4;
    const long e = t0 + (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (e < n && blockIdx.x * blockDim.x + threadIdx.x < 4) {
        float vv[NR];
        float s = 0.f;
#pragma unroll
        for (int k = 0; k < NR; ++k)
            if (k < n_rep) { vv[k] = reps.p[k][e]; s += vv[k]; }
        const float vbar = s / inv_div;
#pragma unroll
        for (int k = 0; k < NR; ++k)
            if (k < n_rep) reps.p[k][e] = reread(reps.p[k] + e) + (vbar - vv[k]);
    }
}

template <int U>
static void launch_average_u(const RepPtrs& reps, int n_rep, long n, hipStream_t st) {
    long b = (n / 4 + (long)kAvgThreads * U - 1) / ((long)kAvgThreads * U);
    if (b < 1) b = 1;
    if (b > kAvgMaxBlocks) b = kAvgMaxBlocks;
    const dim3 grid((unsigned)b), block(kAvgThreads);
    if (n_rep <= 2) launch(average_k<2, U>, grid, block, 0, st, reps, n_rep, n);
    else if (n_rep <= 4) launch(average_k<4, U>, grid, block, 0, st, reps, n_rep, n);
    else if (n_rep <= 8) launch(average_k<8, U>, grid, block, 0, st, reps, n_rep, n);
    else launch(average_k<16, U>, grid, block, 0, st, reps, n_rep, n);
}

hipError_t launch_average(const RepPtrs& reps, int n_rep, long n, hipStream_t st) {
    launch_average_u<1>(reps, n_rep, n, st);
    return hipGetLastError();
}

}  // namespace lpp
