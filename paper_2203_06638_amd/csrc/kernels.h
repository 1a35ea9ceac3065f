// kernels.h -- launchers of the gfx950 kernels used by the runtime.
// Every launcher enqueues on `st` and returns hipGetLastError() of the launch.
#pragma once
#include <hip/hip_runtime.h>
#include <cstdint>

namespace lpp {

// Geometry of an implicit-GEMM convolution pass.
//   forward : output pixels (Nb, Ho, Wo) x Ncols = Cout, source = conv input
//             (Nb, Hs, Ws, Cs = padded Cin), B = W_f[Cout][R][S][Cs]
//   dgrad   : output pixels (Nb, Ho, Wo) = conv input grid, Ncols = Cin,
//             source = dY (Nb, Hs, Ws, Cs = Cout), B = W_d[Cin][R][S][Cout]
struct ConvGeom {
    int Nb, Hs, Ws, Cs;   // source activation (NHWC)
    int Ho, Wo, Ncols;    // output grid and channels (NHWC)
    int R, S, stride, pad;
};

enum ConvMode { CONV_FWD = 0, CONV_DGRAD = 1 };

// Y[m][n] (+)= sum_k A[m][k] B[n][k] (+ bias[n]); see ConvGeom.
hipError_t launch_conv_igemm(int mode, const float* src, const float* B, const float* bias, float* Y,
                             const ConvGeom& g, bool accumulate, hipStream_t st);

// Weight gradient: part[split][Cout][Ktot] = partial sums over pixel ranges
// of dY[p][cout] * im2col(X)[p][(r,s,c)].  Returns the number of splits used
// via *splits (computed by wgrad_plan).
struct WgradPlan { int tm, tn, splits, pix_per_split; long part_floats; };
WgradPlan wgrad_plan(int Cout, int Ktot, long M);
hipError_t launch_conv_wgrad(const float* dY, const float* X, float* part, int Nb, int Hi, int Wi, int Cin_p,
                             int Ho, int Wo, int Cout, int R, int S, int stride, int pad, const WgradPlan& p,
                             hipStream_t st);
// Sums the split partials in order and writes the canonical gradient
// g[((cout*Cin + c)*R + r)*S + s] for c < Cin.
hipError_t launch_wgrad_reduce(const float* part, int splits, int Cout, int Ktot, int Cin, int Cin_p, int R, int S,
                               float* g, hipStream_t st);

// Per-channel reductions over an [M][C] NHWC matrix, in two fixed-order
// stages (partials per workgroup in fp64, then a finalize).
int chan_reduce_blocks(long M, int C);
// stats: psum[b][c] = sum x, psq[b][c] = sum x^2 over the block's rows
hipError_t launch_bn_stats_partial(const float* x, long M, int C, double* psum, double* psq, hipStream_t st);
// mean, rstd, and the affine apply coefficients scale = gamma*rstd,
// shift = beta - mean*scale
hipError_t launch_bn_stats_finalize(const double* psum, const double* psq, int nblk, long M, int C,
                                    const float* gamma, const float* beta, float eps, float* mean, float* rstd,
                                    float* scale, float* shift, hipStream_t st);
hipError_t launch_chan_affine(const float* x, const float* scale, const float* shift, float* y, long M, int C,
                              hipStream_t st);
// backward sums: psum[b][c] = sum dy, psq[b][c] = sum dy * (x - mean) * rstd
hipError_t launch_bn_bwd_partial(const float* dy, const float* x, const float* mean, const float* rstd, long M,
                                 int C, double* psum, double* psq, hipStream_t st);
// dbeta = sum dy, dgamma = sum dy*xhat (written to g_gamma/g_beta if not
// null), and the data-gradient coefficients a = gamma*rstd, mdy = sum dy / M,
// mdyx = sum dy*xhat / M
hipError_t launch_bn_bwd_finalize(const double* psum, const double* psq, int nblk, long M, int C,
                                  const float* gamma, const float* rstd, float* g_gamma, float* g_beta,
                                  float* coef_a, float* coef_mdy, float* coef_mdyx, hipStream_t st);
// dx (+)= a*(dy - mdy - (x - mean)*rstd*mdyx)
hipError_t launch_bn_bwd_data(const float* dy, const float* x, const float* mean, const float* rstd,
                              const float* a, const float* mdy, const float* mdyx, float* dx, long M, int C,
                              bool accumulate, hipStream_t st);
// column sums of dy (conv bias gradient): out[c] = sum_m dy[m][c]
hipError_t launch_col_sum_partial(const float* dy, long M, int C, double* psum, hipStream_t st);
hipError_t launch_col_sum_finalize(const double* psum, int nblk, int C, float* out, hipStream_t st);

// elementwise (n multiple of 4)
hipError_t launch_relu_fwd(const float* x, float* y, long n, hipStream_t st);
hipError_t launch_relu_bwd(const float* dy, const float* x, float* dx, long n, bool accumulate, hipStream_t st);
hipError_t launch_add_fwd(const float* a, const float* b, float* y, long n, hipStream_t st);
hipError_t launch_copy_acc(const float* src, float* dst, long n, bool accumulate, hipStream_t st);

hipError_t launch_maxpool_fwd(const float* x, float* y, uint8_t* arg, int Nb, int H, int W, int C, int Ho, int Wo,
                              int k, int stride, int pad, hipStream_t st);
hipError_t launch_maxpool_bwd(const float* dy, const uint8_t* arg, float* dx, int Nb, int H, int W, int C, int Ho,
                              int Wo, int k, int stride, int pad, bool accumulate, hipStream_t st);
hipError_t launch_gap_fwd(const float* x, float* y, int Nb, int HW, int C, hipStream_t st);
hipError_t launch_gap_bwd(const float* dy, float* dx, int Nb, int HW, int C, bool accumulate, hipStream_t st);
hipError_t launch_linear_fwd(const float* x, const float* W, const float* b, float* y, int Nb, int I, int O,
                             hipStream_t st);
hipError_t launch_linear_bwd_w(const float* dz, const float* x, float* gW, float* gb, int Nb, int I, int O,
                               hipStream_t st);
hipError_t launch_linear_bwd_x(const float* dz, const float* W, float* dx, int Nb, int I, int O, bool accumulate,
                               hipStream_t st);
// mean softmax cross-entropy: loss[0], dz = (softmax - onehot)/N
hipError_t launch_softmax_ce(const float* z, const int* labels, float* dz, float* loss, int Nb, int Cls,
                             hipStream_t st);

// NCHW (C channels) -> NHWC (Cp >= C channels, zero-padded)
hipError_t launch_nchw_to_nhwc(const float* src, float* dst, int Nb, int C, int H, int W, int Cp, hipStream_t st);
// NHWC (Cp) -> NCHW (C), for inspection
hipError_t launch_nhwc_to_nchw(const float* src, float* dst, int Nb, int C, int H, int W, int Cp, hipStream_t st);

// Snapshot of the shared replica (Alg. 1: lock-free read of every entry):
// v[e] = x[e] for e < d, and each conv weight also into its forward layout
// W_f[cout][r][s][cin_p] and dgrad layout W_d[cin][r][s][cout].
struct SnapConv { long src, n; int cout, cin, cin_p, R, S; long dst_f, dst_d; };
hipError_t launch_snapshot(const float* x, float* v, long d, const SnapConv* convs_dev, int n_convs, float* wbase,
                           hipStream_t st);

// Block update (Alg. 1 updater's last step), e in [lo, hi):
//   m = mu*m + g + wd*x; x -= lr*m   (m == null: x -= lr*(g + wd*x))
hipError_t launch_sgd_update(float* x, float* m, const float* g, long lo, long hi, float lr, float mu, float wd,
                             hipStream_t st);
// Averaging round (Alg. 1 averager) over n_rep replicas of n floats.
constexpr int kMaxReplicas = 16;
struct RepPtrs { float* p[kMaxReplicas]; };
hipError_t launch_average(const RepPtrs& reps, int n_rep, long n, hipStream_t st);

}  // namespace lpp
