// misc_f32.hip -- the non-convolution kernels of the step: batch-norm
// statistics / apply / backward, ReLU, residual add, max pool, global
// average pool, the linear head, softmax cross-entropy, layout conversions,
// the replica snapshot, the block SGD update and replica averaging.
//
// Activations are NHWC float32.  Channel reductions run in two fixed-order
// stages (per-workgroup fp64 partials, then one pass over the partials), so
// every result is bitwise reproducible run to run.
#include "kernels.h"

namespace lpp {

typedef float f4 __attribute__((ext_vector_type(4)));

static inline unsigned nblocks(long n, int per) { return (unsigned)((n + per - 1) / per); }

// ------------------------------------------------------------------------
// per-channel reductions over [M][C]
// ------------------------------------------------------------------------

constexpr int kRedRows = 1024;   // rows of the matrix per reduction workgroup

int chan_reduce_blocks(long M, int C) {
    (void)C;
    return (int)((M + kRedRows - 1) / kRedRows);
}

// KIND 0: (sum x, sum x^2)   KIND 1: (sum dy, sum dy*xhat)   KIND 2: sum dy
template <int KIND>
__global__ __launch_bounds__(256) void chan_partial(const float* __restrict__ a, const float* __restrict__ b,
                                                    const float* __restrict__ mean, const float* __restrict__ rstd,
                                                    long M, int C, double* __restrict__ p0, double* __restrict__ p1) {
    __shared__ double s0[256], s1[256];
    const int C4 = C >> 2;
    const int tid = threadIdx.x;
    const long r0 = (long)blockIdx.x * kRedRows;
    const long r1 = min(M, r0 + kRedRows);
    // threads tile (row lanes) x (channel quads); quads beyond 256 loop
    for (int qbase = 0; qbase < C4; qbase += 256) {
        const int nq = min(256, C4 - qbase);
        const int rl = 256 / nq;             // rows processed in parallel
        const int q = qbase + tid % nq;
        const int lr = tid / nq;
        double x0[4] = {0, 0, 0, 0}, x1[4] = {0, 0, 0, 0};
        float mu[4] = {0, 0, 0, 0}, rs[4] = {0, 0, 0, 0};
        if (KIND == 1 && lr < rl) {
#pragma unroll
            for (int i = 0; i < 4; ++i) { mu[i] = mean[q * 4 + i]; rs[i] = rstd[q * 4 + i]; }
        }
        if (lr < rl) {
            for (long r = r0 + lr; r < r1; r += rl) {
                const f4 va = *(const f4*)(a + r * C + q * 4);
                if (KIND == 0) {
#pragma unroll
                    for (int i = 0; i < 4; ++i) { x0[i] += (double)va[i]; x1[i] += (double)va[i] * (double)va[i]; }
                } else if (KIND == 1) {
                    const f4 vb = *(const f4*)(b + r * C + q * 4);
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        x0[i] += (double)va[i];
                        x1[i] += (double)va[i] * (double)((vb[i] - mu[i]) * rs[i]);
                    }
                } else {
#pragma unroll
                    for (int i = 0; i < 4; ++i) x0[i] += (double)va[i];
                }
            }
        }
        // reduce over the row lanes, one channel component at a time, fixed order
        for (int i = 0; i < 4; ++i) {
            s0[tid] = x0[i];
            s1[tid] = x1[i];
            __syncthreads();
            if (tid < nq) {
                double t0 = 0.0, t1 = 0.0;
                for (int l = 0; l < rl; ++l) { t0 += s0[l * nq + tid]; t1 += s1[l * nq + tid]; }
                const long o = (long)blockIdx.x * C + (qbase + tid) * 4 + i;
                p0[o] = t0;
                if (KIND != 2) p1[o] = t1;
            }
            __syncthreads();
        }
    }
}

__global__ void bn_stats_finalize_k(const double* __restrict__ psum, const double* __restrict__ psq, int nblk, long M,
                                    int C, const float* __restrict__ gamma, const float* __restrict__ beta, float eps,
                                    float* mean, float* rstd, float* scale, float* shift) {
    const int c = blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= C) return;
    double s = 0.0, q = 0.0;
    for (int b = 0; b < nblk; ++b) { s += psum[(long)b * C + c]; q += psq[(long)b * C + c]; }
    const double mu = s / (double)M;
    double var = q / (double)M - mu * mu;
    if (var < 0.0) var = 0.0;
    const double r = 1.0 / sqrt(var + (double)eps);
    mean[c] = (float)mu;
    rstd[c] = (float)r;
    const double sc = (double)gamma[c] * r;
    scale[c] = (float)sc;
    shift[c] = (float)((double)beta[c] - mu * sc);
}

__global__ void bn_bwd_finalize_k(const double* __restrict__ psum, const double* __restrict__ psq, int nblk, long M,
                                  int C, const float* __restrict__ gamma, const float* __restrict__ rstd,
                                  float* g_gamma, float* g_beta, float* ca, float* cmdy, float* cmdyx) {
    const int c = blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= C) return;
    double s = 0.0, q = 0.0;
    for (int b = 0; b < nblk; ++b) { s += psum[(long)b * C + c]; q += psq[(long)b * C + c]; }
    if (g_gamma) g_gamma[c] = (float)q;
    if (g_beta) g_beta[c] = (float)s;
    ca[c] = gamma[c] * rstd[c];
    cmdy[c] = (float)(s / (double)M);
    cmdyx[c] = (float)(q / (double)M);
}

__global__ void col_sum_finalize_k(const double* __restrict__ psum, int nblk, int C, float* out) {
    const int c = blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= C) return;
    double s = 0.0;
    for (int b = 0; b < nblk; ++b) s += psum[(long)b * C + c];
    out[c] = (float)s;
}

hipError_t launch_bn_stats_partial(const float* x, long M, int C, double* psum, double* psq, hipStream_t st) {
    hipLaunchKernelGGL(chan_partial<0>, dim3(chan_reduce_blocks(M, C)), dim3(256), 0, st, x, nullptr, nullptr,
                       nullptr, M, C, psum, psq);
    return hipGetLastError();
}
hipError_t launch_bn_stats_finalize(const double* psum, const double* psq, int nblk, long M, int C,
                                    const float* gamma, const float* beta, float eps, float* mean, float* rstd,
                                    float* scale, float* shift, hipStream_t st) {
    hipLaunchKernelGGL(bn_stats_finalize_k, dim3(nblocks(C, 64)), dim3(64), 0, st, psum, psq, nblk, M, C, gamma,
                       beta, eps, mean, rstd, scale, shift);
    return hipGetLastError();
}
hipError_t launch_bn_bwd_partial(const float* dy, const float* x, const float* mean, const float* rstd, long M,
                                 int C, double* psum, double* psq, hipStream_t st) {
    hipLaunchKernelGGL(chan_partial<1>, dim3(chan_reduce_blocks(M, C)), dim3(256), 0, st, dy, x, mean, rstd, M, C,
                       psum, psq);
    return hipGetLastError();
}
hipError_t launch_bn_bwd_finalize(const double* psum, const double* psq, int nblk, long M, int C,
                                  const float* gamma, const float* rstd, float* g_gamma, float* g_beta,
                                  float* coef_a, float* coef_mdy, float* coef_mdyx, hipStream_t st) {
    hipLaunchKernelGGL(bn_bwd_finalize_k, dim3(nblocks(C, 64)), dim3(64), 0, st, psum, psq, nblk, M, C, gamma, rstd,
                       g_gamma, g_beta, coef_a, coef_mdy, coef_mdyx);
    return hipGetLastError();
}
hipError_t launch_col_sum_partial(const float* dy, long M, int C, double* psum, hipStream_t st) {
    hipLaunchKernelGGL(chan_partial<2>, dim3(chan_reduce_blocks(M, C)), dim3(256), 0, st, dy, nullptr, nullptr,
                       nullptr, M, C, psum, nullptr);
    return hipGetLastError();
}
hipError_t launch_col_sum_finalize(const double* psum, int nblk, int C, float* out, hipStream_t st) {
    hipLaunchKernelGGL(col_sum_finalize_k, dim3(nblocks(C, 64)), dim3(64), 0, st, psum, nblk, C, out);
    return hipGetLastError();
}

// ------------------------------------------------------------------------
// elementwise
// ------------------------------------------------------------------------

__global__ void chan_affine_k(const f4* __restrict__ x, const float* __restrict__ scale,
                              const float* __restrict__ shift, f4* __restrict__ y, long n4, int C) {
    for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += (long)gridDim.x * blockDim.x) {
        const int c = (int)((i * 4) % C);
        f4 v = x[i];
        f4 o;
#pragma unroll
        for (int k = 0; k < 4; ++k) o[k] = v[k] * scale[c + k] + shift[c + k];
        y[i] = o;
    }
}

__global__ void bn_bwd_data_k(const f4* __restrict__ dy, const f4* __restrict__ x, const float* __restrict__ mean,
                              const float* __restrict__ rstd, const float* __restrict__ ca,
                              const float* __restrict__ cmdy, const float* __restrict__ cmdyx, f4* __restrict__ dx,
                              long n4, int C, int acc) {
    for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += (long)gridDim.x * blockDim.x) {
        const int c = (int)((i * 4) % C);
        f4 g = dy[i], v = x[i];
        f4 o = acc ? dx[i] : f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const float xh = (v[k] - mean[c + k]) * rstd[c + k];
            o[k] += ca[c + k] * (g[k] - cmdy[c + k] - xh * cmdyx[c + k]);
        }
        dx[i] = o;
    }
}

__global__ void relu_fwd_k(const f4* __restrict__ x, f4* __restrict__ y, long n4) {
    for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += (long)gridDim.x * blockDim.x) {
        f4 v = x[i];
#pragma unroll
        for (int k = 0; k < 4; ++k) v[k] = v[k] > 0.f ? v[k] : 0.f;
        y[i] = v;
    }
}

__global__ void relu_bwd_k(const f4* __restrict__ dy, const f4* __restrict__ x, f4* __restrict__ dx, long n4,
                           int acc) {
    for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += (long)gridDim.x * blockDim.x) {
        f4 g = dy[i], v = x[i];
        f4 o = acc ? dx[i] : f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int k = 0; k < 4; ++k) o[k] += v[k] > 0.f ? g[k] : 0.f;
        dx[i] = o;
    }
}

__global__ void add_fwd_k(const f4* __restrict__ a, const f4* __restrict__ b, f4* __restrict__ y, long n4) {
    for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += (long)gridDim.x * blockDim.x)
        y[i] = a[i] + b[i];
}

__global__ void copy_acc_k(const f4* __restrict__ s, f4* __restrict__ d, long n4, int acc) {
    for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += (long)gridDim.x * blockDim.x)
        d[i] = acc ? d[i] + s[i] : s[i];
}

static unsigned ew_grid(long n4) {
    long b = (n4 + 255) / 256;
    return (unsigned)(b < 8192 ? (b < 1 ? 1 : b) : 8192);
}

hipError_t launch_chan_affine(const float* x, const float* scale, const float* shift, float* y, long M, int C,
                              hipStream_t st) {
    const long n4 = M * C / 4;
    hipLaunchKernelGGL(chan_affine_k, dim3(ew_grid(n4)), dim3(256), 0, st, (const f4*)x, scale, shift, (f4*)y, n4,
                       C);
    return hipGetLastError();
}
hipError_t launch_bn_bwd_data(const float* dy, const float* x, const float* mean, const float* rstd,
                              const float* a, const float* mdy, const float* mdyx, float* dx, long M, int C,
                              bool accumulate, hipStream_t st) {
    const long n4 = M * C / 4;
    hipLaunchKernelGGL(bn_bwd_data_k, dim3(ew_grid(n4)), dim3(256), 0, st, (const f4*)dy, (const f4*)x, mean, rstd,
                       a, mdy, mdyx, (f4*)dx, n4, C, (int)accumulate);
    return hipGetLastError();
}
hipError_t launch_relu_fwd(const float* x, float* y, long n, hipStream_t st) {
    hipLaunchKernelGGL(relu_fwd_k, dim3(ew_grid(n / 4)), dim3(256), 0, st, (const f4*)x, (f4*)y, n / 4);
    return hipGetLastError();
}
hipError_t launch_relu_bwd(const float* dy, const float* x, float* dx, long n, bool accumulate, hipStream_t st) {
    hipLaunchKernelGGL(relu_bwd_k, dim3(ew_grid(n / 4)), dim3(256), 0, st, (const f4*)dy, (const f4*)x, (f4*)dx,
                       n / 4, (int)accumulate);
    return hipGetLastError();
}
hipError_t launch_add_fwd(const float* a, const float* b, float* y, long n, hipStream_t st) {
    hipLaunchKernelGGL(add_fwd_k, dim3(ew_grid(n / 4)), dim3(256), 0, st, (const f4*)a, (const f4*)b, (f4*)y,
                       n / 4);
    return hipGetLastError();
}
hipError_t launch_copy_acc(const float* src, float* dst, long n, bool accumulate, hipStream_t st) {
    hipLaunchKernelGGL(copy_acc_k, dim3(ew_grid(n / 4)), dim3(256), 0, st, (const f4*)src, (f4*)dst, n / 4,
                       (int)accumulate);
    return hipGetLastError();
}

// ------------------------------------------------------------------------
// pooling
// ------------------------------------------------------------------------

// arg holds the winning tap r*k + s (first maximum in row-major scan order)
__global__ void maxpool_fwd_k(const float* __restrict__ x, float* __restrict__ y, uint8_t* __restrict__ arg,
                              int Nb, int H, int W, int C, int Ho, int Wo, int k, int st, int pad) {
    const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
    const long total = (long)Nb * Ho * Wo * C;
    if (idx >= total) return;
    const int c = (int)(idx % C);
    long t = idx / C;
    const int q = (int)(t % Wo);
    t /= Wo;
    const int p = (int)(t % Ho);
    const int n = (int)(t / Ho);
    float m = -INFINITY;
    int am = 0;
    for (int r = 0; r < k; ++r) {
        const int hi = p * st - pad + r;
        if (hi < 0 || hi >= H) continue;
        for (int s = 0; s < k; ++s) {
            const int wi = q * st - pad + s;
            if (wi < 0 || wi >= W) continue;
            const float v = x[(((long)n * H + hi) * W + wi) * C + c];
            if (v > m) { m = v; am = r * k + s; }
        }
    }
    y[idx] = m;
    arg[idx] = (uint8_t)am;
}

__global__ void maxpool_bwd_k(const float* __restrict__ dy, const uint8_t* __restrict__ arg, float* __restrict__ dx,
                              int Nb, int H, int W, int C, int Ho, int Wo, int k, int st, int pad, int acc) {
    const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
    const long total = (long)Nb * H * W * C;
    if (idx >= total) return;
    const int c = (int)(idx % C);
    long t = idx / C;
    const int w = (int)(t % W);
    t /= W;
    const int h = (int)(t % H);
    const int n = (int)(t / H);
    float s = 0.f;
    // windows p with p*st - pad <= h <= p*st - pad + k - 1
    const int p_lo = max(0, (h + pad - k + st) / st), p_hi = min(Ho - 1, (h + pad) / st);
    const int q_lo = max(0, (w + pad - k + st) / st), q_hi = min(Wo - 1, (w + pad) / st);
    for (int p = p_lo; p <= p_hi; ++p)
        for (int q = q_lo; q <= q_hi; ++q) {
            const int r = h - (p * st - pad), ss = w - (q * st - pad);
            if (r < 0 || r >= k || ss < 0 || ss >= k) continue;
            const long o = (((long)n * Ho + p) * Wo + q) * C + c;
            if (arg[o] == r * k + ss) s += dy[o];
        }
    dx[idx] = acc ? dx[idx] + s : s;
}

__global__ void gap_fwd_k(const float* __restrict__ x, float* __restrict__ y, int Nb, int HW, int C) {
    const int idx = blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= Nb * C) return;
    const int n = idx / C, c = idx - n * C;
    float s = 0.f;
    for (int e = 0; e < HW; ++e) s += x[((long)n * HW + e) * C + c];
    y[idx] = s / (float)HW;
}

__global__ void gap_bwd_k(const float* __restrict__ dy, float* __restrict__ dx, int Nb, int HW, int C, int acc) {
    const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= (long)Nb * HW * C) return;
    const int c = (int)(idx % C);
    const int n = (int)(idx / ((long)HW * C));
    const float v = dy[n * C + c] / (float)HW;
    dx[idx] = acc ? dx[idx] + v : v;
}

hipError_t launch_maxpool_fwd(const float* x, float* y, uint8_t* arg, int Nb, int H, int W, int C, int Ho, int Wo,
                              int k, int stride, int pad, hipStream_t st) {
    const long total = (long)Nb * Ho * Wo * C;
    hipLaunchKernelGGL(maxpool_fwd_k, dim3(nblocks(total, 256)), dim3(256), 0, st, x, y, arg, Nb, H, W, C, Ho, Wo, k,
                       stride, pad);
    return hipGetLastError();
}
hipError_t launch_maxpool_bwd(const float* dy, const uint8_t* arg, float* dx, int Nb, int H, int W, int C, int Ho,
                              int Wo, int k, int stride, int pad, bool accumulate, hipStream_t st) {
    const long total = (long)Nb * H * W * C;
    hipLaunchKernelGGL(maxpool_bwd_k, dim3(nblocks(total, 256)), dim3(256), 0, st, dy, arg, dx, Nb, H, W, C, Ho, Wo,
                       k, stride, pad, (int)accumulate);
    return hipGetLastError();
}
hipError_t launch_gap_fwd(const float* x, float* y, int Nb, int HW, int C, hipStream_t st) {
    hipLaunchKernelGGL(gap_fwd_k, dim3(nblocks((long)Nb * C, 256)), dim3(256), 0, st, x, y, Nb, HW, C);
    return hipGetLastError();
}
hipError_t launch_gap_bwd(const float* dy, float* dx, int Nb, int HW, int C, bool accumulate, hipStream_t st) {
    hipLaunchKernelGGL(gap_bwd_k, dim3(nblocks((long)Nb * HW * C, 256)), dim3(256), 0, st, dy, dx, Nb, HW, C,
                       (int)accumulate);
    return hipGetLastError();
}

// ------------------------------------------------------------------------
// linear head and loss
// ------------------------------------------------------------------------

__global__ void linear_fwd_k(const float* __restrict__ x, const float* __restrict__ W, const float* __restrict__ b,
                             float* __restrict__ y, int Nb, int I, int O) {
    const int idx = blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= Nb * O) return;
    const int n = idx / O, o = idx - n * O;
    float s = b ? b[o] : 0.f;
    for (int i = 0; i < I; ++i) s += W[(long)o * I + i] * x[(long)n * I + i];
    y[idx] = s;
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

// One workgroup; wave w handles samples w, w+4, ...; the batch mean is
// summed by one thread in sample order.
__global__ __launch_bounds__(256) void softmax_ce_k(const float* __restrict__ z, const int* __restrict__ labels,
                                                    float* __restrict__ dz, float* __restrict__ loss,
                                                    float* __restrict__ per_sample, int Nb, int Cls) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    for (int n = wave; n < Nb; n += 4) {
        const float* zr = z + (long)n * Cls;
        float mx = -INFINITY;
        for (int j = lane; j < Cls; j += 64) mx = fmaxf(mx, zr[j]);
        for (int off = 32; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
        float se = 0.f;
        for (int j = lane; j < Cls; j += 64) se += expf(zr[j] - mx);
        for (int off = 32; off > 0; off >>= 1) se += __shfl_xor(se, off);
        const float lse = mx + logf(se);
        const int y = labels[n];
        for (int j = lane; j < Cls; j += 64)
            dz[(long)n * Cls + j] = (expf(zr[j] - lse) - (j == y ? 1.f : 0.f)) / (float)Nb;
        if (lane == 0) per_sample[n] = lse - zr[y];
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        float s = 0.f;
        for (int n = 0; n < Nb; ++n) s += per_sample[n];
        loss[0] = s / (float)Nb;
    }
}

hipError_t launch_linear_fwd(const float* x, const float* W, const float* b, float* y, int Nb, int I, int O,
                             hipStream_t st) {
    hipLaunchKernelGGL(linear_fwd_k, dim3(nblocks((long)Nb * O, 256)), dim3(256), 0, st, x, W, b, y, Nb, I, O);
    return hipGetLastError();
}
hipError_t launch_linear_bwd_w(const float* dz, const float* x, float* gW, float* gb, int Nb, int I, int O,
                               hipStream_t st) {
    hipLaunchKernelGGL(linear_bwd_w_k, dim3(nblocks((long)O * I + O, 256)), dim3(256), 0, st, dz, x, gW, gb, Nb, I,
                       O);
    return hipGetLastError();
}
hipError_t launch_linear_bwd_x(const float* dz, const float* W, float* dx, int Nb, int I, int O, bool accumulate,
                               hipStream_t st) {
    hipLaunchKernelGGL(linear_bwd_x_k, dim3(nblocks((long)Nb * I, 256)), dim3(256), 0, st, dz, W, dx, Nb, I, O,
                       (int)accumulate);
    return hipGetLastError();
}
hipError_t launch_softmax_ce(const float* z, const int* labels, float* dz, float* loss, int Nb, int Cls,
                             hipStream_t st) {
    // per-sample losses live just after the loss scalar (caller sizes loss to 1 + Nb floats)
    hipLaunchKernelGGL(softmax_ce_k, dim3(1), dim3(256), 0, st, z, labels, dz, loss, loss + 1, Nb, Cls);
    return hipGetLastError();
}

// ------------------------------------------------------------------------
// layouts
// ------------------------------------------------------------------------

__global__ void nchw_to_nhwc_k(const float* __restrict__ s, float* __restrict__ d, int Nb, int C, int H, int W,
                               int Cp) {
    const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
    const long total = (long)Nb * H * W * Cp;
    if (idx >= total) return;
    const int c = (int)(idx % Cp);
    const long pix = idx / Cp;
    const int w = (int)(pix % W);
    const long t = pix / W;
    const int h = (int)(t % H);
    const int n = (int)(t / H);
    d[idx] = c < C ? s[(((long)n * C + c) * H + h) * W + w] : 0.f;
}

__global__ void nhwc_to_nchw_k(const float* __restrict__ s, float* __restrict__ d, int Nb, int C, int H, int W,
                               int Cp) {
    const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
    const long total = (long)Nb * C * H * W;
    if (idx >= total) return;
    const int w = (int)(idx % W);
    long t = idx / W;
    const int h = (int)(t % H);
    t /= H;
    const int c = (int)(t % C);
    const int n = (int)(t / C);
    d[idx] = s[(((long)n * H + h) * W + w) * Cp + c];
}

hipError_t launch_nchw_to_nhwc(const float* src, float* dst, int Nb, int C, int H, int W, int Cp, hipStream_t st) {
    const long total = (long)Nb * H * W * Cp;
    hipLaunchKernelGGL(nchw_to_nhwc_k, dim3(nblocks(total, 256)), dim3(256), 0, st, src, dst, Nb, C, H, W, Cp);
    return hipGetLastError();
}
hipError_t launch_nhwc_to_nchw(const float* src, float* dst, int Nb, int C, int H, int W, int Cp, hipStream_t st) {
    const long total = (long)Nb * H * W * C;
    hipLaunchKernelGGL(nhwc_to_nchw_k, dim3(nblocks(total, 256)), dim3(256), 0, st, src, dst, Nb, C, H, W, Cp);
    return hipGetLastError();
}

// ------------------------------------------------------------------------
// snapshot, block update, averaging
// ------------------------------------------------------------------------

__global__ void snapshot_k(const float* __restrict__ x, float* __restrict__ v, long d,
                           const SnapConv* __restrict__ convs, int nc, float* __restrict__ wbase) {
    for (long e = (long)blockIdx.x * blockDim.x + threadIdx.x; e < d; e += (long)gridDim.x * blockDim.x) {
        const float val = x[e];
        v[e] = val;
        // conv segments are sorted by src; find the last with src <= e
        int lo = 0, hi = nc - 1, f = -1;
        while (lo <= hi) {
            const int mid = (lo + hi) >> 1;
            if (convs[mid].src <= e) { f = mid; lo = mid + 1; } else hi = mid - 1;
        }
        if (f < 0) continue;
        const SnapConv cv = convs[f];
        const long o = e - cv.src;
        if (o >= (long)cv.cout * cv.cin * cv.R * cv.S) continue;   // bias / beyond the weight
        const int s = (int)(o % cv.S);
        long t = o / cv.S;
        const int r = (int)(t % cv.R);
        t /= cv.R;
        const int c = (int)(t % cv.cin);
        const int k = (int)(t / cv.cin);
        wbase[cv.dst_f + (((long)k * cv.R + r) * cv.S + s) * cv.cin_p + c] = val;
        wbase[cv.dst_d + (((long)c * cv.R + r) * cv.S + s) * cv.cout + k] = val;
    }
}

hipError_t launch_snapshot(const float* x, float* v, long d, const SnapConv* convs_dev, int n_convs, float* wbase,
                           hipStream_t st) {
    long b = (d + 255) / 256;
    if (b > 16384) b = 16384;
    hipLaunchKernelGGL(snapshot_k, dim3((unsigned)b), dim3(256), 0, st, x, v, d, convs_dev, n_convs, wbase);
    return hipGetLastError();
}

// Each thread owns an aligned quad [4t, 4t+4) of the index space shifted to
// the aligned start below lo; whole quads use 16-byte accesses.
__global__ void sgd_update_k(float* __restrict__ x, float* __restrict__ m, const float* __restrict__ g, long lo,
                             long hi, float lr, float mu, float wd) {
    const long base = lo & ~3L;
    const long nq = (hi - base + 3) / 4;
    for (long q = (long)blockIdx.x * blockDim.x + threadIdx.x; q < nq; q += (long)gridDim.x * blockDim.x) {
        const long e0 = base + 4 * q;
        if (e0 >= lo && e0 + 4 <= hi) {
            f4 xv = *(f4*)(x + e0);
            const f4 gv = *(const f4*)(g + e0);
            if (m) {
                f4 mv = *(f4*)(m + e0);
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    mv[k] = mu * mv[k] + (gv[k] + wd * xv[k]);
                    xv[k] -= lr * mv[k];
                }
                *(f4*)(m + e0) = mv;
            } else {
#pragma unroll
                for (int k = 0; k < 4; ++k) xv[k] -= lr * (gv[k] + wd * xv[k]);
            }
            *(f4*)(x + e0) = xv;
        } else {
            for (long e = e0; e < e0 + 4; ++e) {
                if (e < lo || e >= hi) continue;
                float dir = g[e] + wd * x[e];
                if (m) { m[e] = mu * m[e] + dir; dir = m[e]; }
                x[e] -= lr * dir;
            }
        }
    }
}

hipError_t launch_sgd_update(float* x, float* m, const float* g, long lo, long hi, float lr, float mu, float wd,
                             hipStream_t st) {
    if (hi <= lo) return hipSuccess;
    const long nq = (hi - (lo & ~3L) + 3) / 4;
    long b = (nq + 255) / 256;
    if (b > 8192) b = 8192;
    hipLaunchKernelGGL(sgd_update_k, dim3((unsigned)b), dim3(256), 0, st, x, m, g, lo, hi, lr, mu, wd);
    return hipGetLastError();
}

// v_k = x_k[e]; vbar = (sum_k v_k) / n; x_k[e] = x_k[e] (re-read) + (vbar - v_k)
template <int NR>
__global__ void average_k(RepPtrs reps, int n_rep, long n) {
    const long nq = n / 4;
    const float inv_div = (float)n_rep;
    for (long q = (long)blockIdx.x * blockDim.x + threadIdx.x; q < nq; q += (long)gridDim.x * blockDim.x) {
        f4 v[NR];
        f4 s = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int k = 0; k < NR; ++k) {
            if (k < n_rep) {
                v[k] = *(const f4*)(reps.p[k] + 4 * q);
                s += v[k];
            }
        }
        const f4 vbar = s / inv_div;
#pragma unroll
        for (int k = 0; k < NR; ++k) {
            if (k < n_rep) {
                f4* p = (f4*)(reps.p[k] + 4 * q);
                *p = *p + (vbar - v[k]);
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
            if (k < n_rep) reps.p[k][e] = reps.p[k][e] + (vbar - vv[k]);
    }
}

hipError_t launch_average(const RepPtrs& reps, int n_rep, long n, hipStream_t st) {
    long b = (n / 4 + 255) / 256;
    if (b < 1) b = 1;
    if (b > 8192) b = 8192;
    if (n_rep <= 2)
        hipLaunchKernelGGL(average_k<2>, dim3((unsigned)b), dim3(256), 0, st, reps, n_rep, n);
    else if (n_rep <= 4)
        hipLaunchKernelGGL(average_k<4>, dim3((unsigned)b), dim3(256), 0, st, reps, n_rep, n);
    else if (n_rep <= 8)
        hipLaunchKernelGGL(average_k<8>, dim3((unsigned)b), dim3(256), 0, st, reps, n_rep, n);
    else
        hipLaunchKernelGGL(average_k<16>, dim3((unsigned)b), dim3(256), 0, st, reps, n_rep, n);
    return hipGetLastError();
}

}  // namespace lpp
