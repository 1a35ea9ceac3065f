// kernels.h -- launchers of the gfx950 kernels used by the runtime.
// Every launcher enqueues on `st` and returns hipGetLastError() of the launch.
// Launchers that take `int dt` read and write activations stored as DT_F32
// (float) or DT_BF16 (bfloat16 bit patterns, act.h) through void pointers;
// parameters, gradients, batch-norm statistics and the head's features and
// logits are always float32.
#pragma once
#include <hip/hip_runtime.h>
#include <cstdint>

namespace lpp {

enum DType { DT_F32 = 0, DT_BF16 = 1 };

// Geometry of an implicit-GEMM convolution pass.
//   forward : output pixels (Nb, Ho, Wo) x Ncols = Cout, source = conv input
//             (Nb, Hs, Ws, Cs = padded Cin), B = W_f[Cout][R][S][Cs]
//   dgrad   : output pixels (Nb, Ho, Wo) = conv input grid, Ncols = Cin,
//             source = dY (Nb, Hs, Ws, Cs = Cout), B = W_d[Cin][R][S][Cout]
struct ConvGeom {
    int Nb, Hs, Ws, Cs;   // source activation (NHWC)
    int Ho, Wo, Ncols;    // output grid and channels (NHWC)
    int R, S, stride, pad;
    // bf16 passes: the workgroups a pass aims for (the larger tiles are taken
    // while they still give this many); with several worker streams running
    // at once each pass needs only its share of the chip
    int fill = 512;
};

enum ConvMode { CONV_FWD = 0, CONV_DGRAD = 1 };

// Per-step arguments, read by the step's kernels from device memory so that
// one captured graph serves every step of a worker on a partition.
struct StepArgs {
    const float* images;
    const int* labels;
    float lr;
    long trace_slot;   // this step's row of the timestamp log, or -1
};
hipError_t launch_set_step_args(StepArgs* dst, const float* images, const int* labels, float lr, long trace_slot,
                                hipStream_t st);
// Step tracing: one kernel of one thread that stores the device's constant-
// rate clock (wall_clock64, 100 MHz) into log[slot * 4 + k] with slot =
// args->trace_slot (nothing when it is negative); kernels of a stream run in
// order, so a timestamp kernel marks a point between its neighbours.
hipError_t launch_timestamp(unsigned long long* log, const StepArgs* args, long slot, int k, hipStream_t st);

// Where a batch-norm reduction goes.  With acc set, every workgroup adds its
// tile's sums into per-channel fp64 accumulators acc[q][kAccSlots][C] (q
// selects the sum; bnacc.h), merged across workgroups in arrival order; the
// first kernel of a step zeroes them.  Otherwise tile t writes its partials
// to p0..p2 [T][C] and a finalize kernel merges them in a fixed order, so the
// result is bitwise reproducible.  Eight copies per channel (a power of two;
// acc_add picks workgroup b's copy): with 512-workgroup producers 64 adds
// meet at an address, and every consumer workgroup reads 8 per sum.  Measured against
// 1, 2, 4, 16 and 32 copies: 8 is the fastest on ResNet-20 (332K samples/s
// against 316K with 32, 291K with 2) and on every other workload.
constexpr int kAccSlots = 8;
static_assert((kAccSlots & (kAccSlots - 1)) == 0, "kAccSlots must be a power of two");
struct BnSums {
    double* acc;
    float* p0;
    float* p1;
    float* p2;
};

// A training-mode batch norm's coefficients: from the batch sums acc
// [2][kAccSlots][C] (sum y, sum y^2 over M rows) with gamma, beta, eps, or
// -- acc null -- read from aux = [mean | rstd | scale | shift].
struct BnFwd {
    const double* acc;
    const float* gamma;
    const float* beta;
    float eps;
    long M;
    float* aux;
};

// Largest source channel count of a forward pass that folds a BN + ReLU into
// its operand staging.
constexpr int kFoldMaxC = 512;

// Y[m][n] (+)= sum_k A[m][k] B[n][k] (+ bias[n]); see ConvGeom.  Forward
// passes with stats non-null also produce the batch-norm sums of Y: into
// acc, q = 0: sum y and q = 1: sum y^2 (each row tile's share formed from its
// mean and sum of squared deviations); as partials, the tile mean (p0) and
// sum of squared deviations (p1), T = ceil(M / conv_tile_rows(g)) tiles.
// inbn (forward only; see conv_fold_ok): src is the input of a BN + ReLU
// and the pass reads relu(bn(src)) without storing it.
// Data gradients with stats (and bsum): the output g is the gradient at a
// training-mode BN + ReLU whose input x1 has g's layout; the pass also forms
// that BN backward's sums, q = 0: sum gm and q = 1: sum gm*xhat, gm = g
// where fma(x1, scale, shift) > 0, xhat = (x1 - mean) rstd, from aux =
// [mean | rstd | scale | shift]: into stats->acc, or as partials p0/p1 per
// tile, conv_dgrad_sum_tiles(g) tiles (spatial kernel only).  With y
// non-null the ReLU decision is y > 0 instead (y the stored output of a BN +
// residual add + ReLU group), and the pass may accumulate: the sums then
// describe the accumulated gradient.
struct BnBwdSum {
    const float* x1;
    const float* aux;
    const float* y = nullptr;
};
// How a pass writes Y: kStoreSet overwrites, kStoreAdd adds to what Y
// holds, kStoreRelu (forward, without stats) overwrites with max(y, 0) -- a
// ReLU whose input the conv alone produces, fused into its epilogue.
constexpr int kStoreSet = 0, kStoreAdd = 1, kStoreRelu = 2;
hipError_t launch_conv_igemm(int mode, const float* src, const float* B, const float* bias, float* Y,
                             const ConvGeom& g, int store, const BnSums* stats, hipStream_t st,
                             const BnFwd* inbn = nullptr, const BnBwdSum* bsum = nullptr);
// Tiles of the spatial data-gradient kernel for g, or 0 when it does not take g.
int conv_dgrad_sum_tiles(const ConvGeom& g);
int conv_tile_rows(const ConvGeom& g);

// Weight gradient: part[split][Cout][Ktot] = partial sums over pixel ranges
// of dY[p][cout] * im2col(X)[p][(r,s,c)].  wgrad_plan chooses the kernel:
// spatial tiles (tile = 1: a split is a tile of OH rows of one image or of
// `imgs` whole images) or GEMM tiles over ranges of pix_per_split pixels.
struct WgradPlan { int tm, tn, splits, pix_per_split; long part_floats; int tile, oh, imgs; };
WgradPlan wgrad_plan(int Nb, int Hi, int Wi, int Cin_p, int Ho, int Wo, int Cout, int R, int S, int stride, int pad);
// in_ss (spatial-tile plans only): X is the input of a BN + ReLU whose
// scale and shift are in_ss[c] and in_ss[Cin_p + c]; the pass reads
// relu(fma(x, scale, shift)).
hipError_t launch_conv_wgrad(const float* dY, const float* X, float* part, int Nb, int Hi, int Wi, int Cin_p,
                             int Ho, int Wo, int Cout, int R, int S, int stride, int pad, const WgradPlan& p,
                             hipStream_t st, const float* in_ss = nullptr);
// A forward pass with this geometry and weight-gradient plan can fold a
// preceding BN + ReLU (spatial kernels, at most kFoldMaxC source channels).
bool conv_fold_ok(const ConvGeom& g, const WgradPlan& p);
// Split sums of several weight gradients in one launch: job j sums its
// part[split][Cout][Ktot] (16-byte aligned) over the splits and writes the
// canonical gradient g[((cout*Cin + c)*R + r)*S + s] for c < Cin.  Every
// output is summed in an order fixed by its job's split count alone: split
// lane l of L adds splits l, l + L, l + 2L, ... in turn, then the L lane sums
// are combined by a fixed pairwise tree.
constexpr int kWgRedMaxJobs = 16;
struct WgRedJob {
    const float* part;
    float* g;
    int splits, Cout, Ktot, Cin, Cin_p, RS;   // RS = R * S taps
    int lanes_log2;   // L = 2^lanes_log2 split lanes, 1024 / L output quads per workgroup
    int wg0;          // the job's first workgroup
};
struct WgRedTable { WgRedJob job[kWgRedMaxJobs]; int n, wgs; };
// appends a job (false when the table is full or the shapes are not
// reducible in quads)
bool wgred_add(WgRedTable& t, const float* part, int splits, int Cout, int Ktot, int Cin, int Cin_p, int R, int S,
               float* g);
hipError_t launch_wgrad_reduce_multi(const WgRedTable& t, hipStream_t st);

// ---- bf16 convolution passes (conv_bf16.hip): bf16 source, weights and
// output, float32 accumulation; geometry as for the float32 passes.  The
// forward epilogue's batch-norm sums describe the stored (rounded) output;
// partials come per row tile of conv_bf16_tile_rows(g) rows.  Cs and Ncols
// must be multiples of 8; data gradients of stride 1 or 2.  res (forward,
// not accumulating): a tensor of Y's shape added to the rounded output and
// rounded again (a fused residual add); the sums then describe Y.
hipError_t launch_conv_bf16(int mode, const uint16_t* src, const uint16_t* B, const float* bias, uint16_t* Y,
                            const ConvGeom& g, bool accumulate, const BnSums* stats, hipStream_t st,
                            const uint16_t* res = nullptr);
int conv_bf16_tile_rows(const ConvGeom& g);
bool conv_bf16_supported(int mode, const ConvGeom& g);
// weight gradient from bf16 dY and X into float32 partials part[split][Cout]
// [R*S*Cin_p] (summed by launch_wgrad_reduce_multi); plan.tm / plan.tn hold the
// tile's output channels and columns
WgradPlan wgrad_plan_bf16(int Nb, int Ho, int Wo, int Cin_p, int Cout, int R, int S);
hipError_t launch_conv_wgrad_bf16(const uint16_t* dY, const uint16_t* X, float* part, int Nb, int Hi, int Wi,
                                  int Cin_p, int Ho, int Wo, int Cout, int R, int S, int stride, int pad,
                                  const WgradPlan& p, hipStream_t st);

// ---- batch-norm statistics over [M][C] NHWC rows ----
// row tiles of the stand-alone kernels: stats_rows(M, C) rows each (256, or
// fewer for short tensors), stats_tiles(M, C) of them
int stats_rows(long M, int C);
int stats_tiles(long M, int C);
// per row tile: mean and sum of squared deviations per channel
// into p0 / p1 [T][C], or the tile's share of the batch sums added into
// acc [2][kAccSlots][C] (sum x, sum x^2)
hipError_t launch_stats_partial(int dt, const void* x, long M, int C, const BnSums& out, hipStream_t st);
// merges T tiles of R rows (fp64, fixed order) into aux = [mean | rstd |
// scale | shift]: rstd = 1/sqrt(var + eps) with the biased variance,
// scale = gamma*rstd, shift = beta - mean*scale
hipError_t launch_stats_finalize(const float* pmean, const float* pm2, int T, int R, long M, int C,
                                 const float* gamma, const float* beta, float eps, float* aux, hipStream_t st);
// out[c] = sum_t rows_t * pmean[t][c]: column sums from tile means
hipError_t launch_sum_from_tiles(const float* pmean, int T, int R, long M, int C, float* out, hipStream_t st);
// the same over C columns of partials stored with row stride ld
hipError_t launch_sum_from_tiles_ld(const float* pmean, int ld, int T, int R, long M, int C, float* out,
                                    hipStream_t st);
// A training-mode batch norm as the per-channel map x*scale + shift.  With
// acc set, scale and shift come from the batch sums acc [2][kAccSlots][C]
// over M rows (mean, biased variance, rstd = 1/sqrt(var + eps),
// scale = gamma*rstd, shift = beta - mean*scale) and the kernel's first
// workgroup stores [mean | rstd | scale | shift] into aux; with acc null they
// are read from aux + 2C and aux + 3C.
// y = relu?(bn1(x1) [+ r | + bn2(x2)])  (r: residual tensor; x2: a second
// normalised input, used when both branches of a residual add end in BN)
hipError_t launch_bn_act(int dt, const void* x1, const BnFwd& b1, const void* r, const void* x2, const BnFwd* b2,
                         bool relu, void* y, long M, int C, hipStream_t st);

// Async mode, wide layers: the coefficients derived once per batch norm by a
// kernel of one thread per channel instead of in the prologue of every
// apply workgroup (which re-reads C x kAccSlots sums per workgroup).
// Forward: aux = [mean | rstd | scale | shift] from acc [2][kAccSlots][C].
hipError_t launch_bn_fwd_coef(const BnFwd& b, int C, hipStream_t st);
// workgroups the apply kernels launch for M rows of C channels
int bn_apply_groups(long M, int C);

// ---- batch-norm backward (with the group's ReLU mask and residual fan-out) ----
struct BnBwdArgs {
    const void* dy;                                    // gradient at the group output
    const void* mask;                                  // ReLU output (g = dy where > 0) or null
    const void* x1; const float* mean1; const float* rstd1;    // BN input and statistics
    const void* x2; const float* mean2; const float* rstd2;    // second BN of a dual group, or null
    long M;
    int C;
    const float* mask_ss = nullptr;   // mask null: ReLU decision fma(x1, scale, shift) > 0, scale | shift here
};
// per row tile (stats_rows), the tile's sum g, sum g*xhat1 and sum g*xhat2
// added into acc [3][kAccSlots][C], or written to p0..p2 [T][C]
hipError_t launch_bn_bwd_reduce(int dt, const BnBwdArgs& a, const BnSums& out, hipStream_t st);
// fixed-order merge of T tile partials: gg/gb (dgamma, dbeta; null = not
// wanted) and coef = [gamma*rstd | mean g | mean g*xhat] per channel; the
// second set for a dual group (coef2 null if not)
hipError_t launch_bn_bwd_finalize(const float* p0, const float* p1, const float* p2, int T, long M, int C,
                                  const float* gamma1, const float* rstd1, float* gg1, float* gb1, float* coef1,
                                  const float* gamma2, const float* rstd2, float* gg2, float* gb2, float* coef2,
                                  hipStream_t st);
// Coefficients of the backward apply.  With acc set they are derived in its
// prologue from the sums acc [3][kAccSlots][C]: per batch norm a =
// gamma*rstd, mean g and mean g*xhat, and its first workgroup also stores
// dgamma = sum g*xhat and dbeta = sum g (null pointers: not wanted).
// Otherwise they are read from coef1 / coef2 (written by the finalize).
// Neither: no batch-norm input gradient is formed (only dres).
struct BnBwdCoef {
    const double* acc;
    const float* gamma1; float* gg1; float* gb1;
    const float* gamma2; float* gg2; float* gb2;
    const float* coef1; const float* coef2;
};
// Async mode, wide layers: coef1 (and coef2) = [gamma*rstd | mean g |
// mean g*xhat] and dgamma / dbeta (k.gg*, k.gb*, null = not wanted) from the
// sums k.acc [3][kAccSlots][C], one thread per channel.
hipError_t launch_bn_bwd_coef(const BnBwdArgs& a, const BnBwdCoef& k, float* coef1, float* coef2, hipStream_t st);
// dx = a*(g - mean g - xhat*mean g*xhat) into dx1 / dx2 (null = skip), and g
// into dres (the residual branch) -- each written or accumulated
hipError_t launch_bn_bwd_apply(int dt, const BnBwdArgs& a, const BnBwdCoef& k, void* dx1, bool acc1, void* dx2,
                               bool acc2, void* dres, bool accres, hipStream_t st);

// ---- classifier head: global average pool, linear, softmax CE ----
// Wide heads (C % 16 == 0, C*O >= kHeadWideMin) run as pooling + a matrix-core
// product + softmax; narrow ones as one fused kernel per sample.
constexpr long kHeadWideMin = 16384;
bool head_wide(int C, int O);
hipError_t launch_head_fwd(int dt, const void* x, int Nb, int HW, int C, const float* W, const float* b, int O,
                           const StepArgs* args, float* feat, float* logits, float* dz, float* loss_per,
                           hipStream_t st);
// gW/gb (null: only the loss) and the batch-mean loss
hipError_t launch_head_bwd_w(const float* dz, const float* feat, int Nb, int C, int O, float* gW, float* gb,
                             const float* loss_per, float* loss, hipStream_t st);
// dx (written or accumulated) = (dz W) / HW broadcast over the pixels;
// scratch: Nb*C floats, used by the wide form
hipError_t launch_head_bwd_x(int dt, const float* dz, const float* W, int Nb, int HW, int C, int O, void* dx,
                             bool acc, float* scratch, hipStream_t st);

// elementwise (n multiple of 4)
hipError_t launch_relu_fwd(int dt, const void* x, void* y, long n, hipStream_t st);
hipError_t launch_relu_bwd(int dt, const void* dy, const void* x, void* dx, long n, bool accumulate, hipStream_t st);
// dy (M x C, C a multiple of 4) := dy where y > 0, else 0, in place, y a
// ReLU's stored output; pmean[tile][c] = the tile's mean of the masked
// column c over stats_tiles(M, C) row tiles of stats_rows(M, C) rows.
hipError_t launch_relu_mask_colsum(int dt, void* dy, const void* y, long M, int C, float* pmean, hipStream_t st);
// Backward of y = concat(a, b) over channels where a and b are stored ReLU
// outputs: da / db (null: not wanted) := the slices of dy, zero where ya / yb
// is; pmean (non-null) as launch_relu_mask_colsum's, over C = ca + cb columns.
hipError_t launch_concat_relu_bwd(int dt, const void* dy, const void* ya, const void* yb, void* da, void* db, long M,
                                  int ca, int cb, float* pmean, hipStream_t st);
hipError_t launch_add_fwd(int dt, const void* a, const void* b, void* y, long n, hipStream_t st);
hipError_t launch_copy_acc(int dt, const void* src, void* dst, long n, bool accumulate, hipStream_t st);
// channel concatenation of two NHWC tensors with `rows` pixels (ca, cb
// multiples of 4) and its backward (da / db null when not wanted)
hipError_t launch_concat_fwd(int dt, const void* a, int ca, const void* b, int cb, void* y, long rows,
                             hipStream_t st);
hipError_t launch_concat_bwd(int dt, const void* dy, long rows, int ca, int cb, void* da, bool acc_a, void* db,
                             bool acc_b, hipStream_t st);

hipError_t launch_maxpool_fwd(int dt, const void* x, void* y, uint8_t* arg, int Nb, int H, int W, int C, int Ho,
                              int Wo, int k, int stride, int pad, hipStream_t st);
hipError_t launch_maxpool_bwd(int dt, const void* dy, const uint8_t* arg, void* dx, int Nb, int H, int W, int C,
                              int Ho, int Wo, int k, int stride, int pad, bool accumulate, hipStream_t st);
// pooled features are float32
hipError_t launch_gap_fwd(int dt, const void* x, float* y, int Nb, int HW, int C, hipStream_t st);
hipError_t launch_gap_bwd(int dt, const float* dy, void* dx, int Nb, int HW, int C, bool accumulate, hipStream_t st);
// y = x W^T + b over Nb rows (then max(y, 0) with relu)
hipError_t launch_linear_fwd(const float* x, const float* W, const float* b, float* y, int Nb, int I, int O,
                             hipStream_t st, bool relu = false);
// Weight-gradient partials of y = x W^T + b over M rows in
// linear_wgrad_splits(M) splits of linear_wgrad_rows(M) rows:
// part_w[split][O][I] (the weight) and, when part_b is non-null,
// part_b[split][ceil4(O)] (the bias, zero past O); both reduce with
// wgrad_reduce_multi (R = S = 1).
constexpr int kLinWgMaxSplits = 512;
int linear_wgrad_rows(long M);
int linear_wgrad_splits(long M);
hipError_t launch_linear_wgrad_part(const float* dz, const float* x, float* part_w, float* part_b, int M, int I,
                                    int O, hipStream_t st);
hipError_t launch_linear_bwd_w(const float* dz, const float* x, float* gW, float* gb, int Nb, int I, int O,
                               hipStream_t st);
hipError_t launch_linear_bwd_x(const float* dz, const float* W, float* dx, int Nb, int I, int O, bool accumulate,
                               hipStream_t st);
// mean softmax cross-entropy: loss[0], per-sample losses at loss[1..N],
// dz = (softmax - onehot)/N
hipError_t launch_softmax_ce(const float* z, const StepArgs* args, float* dz, float* loss, int Nb, int Cls,
                             hipStream_t st);

// the step's NCHW images (C channels) -> NHWC (Cp >= C channels, zero-padded);
// also zeroes the step's n_zero reduction accumulators at zero
hipError_t launch_nchw_to_nhwc(int dt, const StepArgs* args, void* dst, int Nb, int C, int H, int W, int Cp,
                               double* zero, long n_zero, hipStream_t st);
// NHWC (Cp) -> NCHW (C) float32, for inspection
hipError_t launch_nhwc_to_nchw(int dt, const void* src, float* dst, int Nb, int C, int H, int W, int Cp,
                               hipStream_t st);

// Snapshot of the shared replica (Alg. 1: lock-free read of every entry).
// Each conv weight W[cout][cin][R][S] (canonical, in x) goes into its forward
// layout W_f[cout][R][S][cin_p] (channels cin..cin_p-1 stay zero) and its
// data-gradient layout W_d[cin][R][S][cout], stored in the activation type
// (the bf16 cast of the mixed-precision workloads); every other parameter
// (batch-norm gamma/beta, biases, linear weights, per-pixel linear convs) is
// copied into v at its canonical index.  Conv weights are not copied into v:
// no kernel reads them there.
//
// The work is a table of entries, each a run of workgroups: a copy entry
// moves [src, src + n) in chunks of kSnapCopy floats, a conv entry covers one
// conv in kt x ct channel tiles (all R*S taps), each transposed through LDS.
struct SnapEntry {
    long src;       // canonical index: first element (copy) or the weight tensor (conv)
    long n;         // copy: elements
    long dst_f;     // conv: W_f base (elements of the activation type)
    long dst_d;     // conv: W_d base
    long tile0;     // first workgroup of this entry
    int kind;       // 0 copy, 1 conv
    int cout, cin, cin_p, RS;
    int kt, ct, nkt;   // conv: tile of kt output x ct input channels; nkt tiles along cout
};
struct SnapConvDesc { long src; int cout, cin, cin_p, R, S; long dst_f, dst_d; };
constexpr int kSnapCopy = 4096;       // floats per copy workgroup
constexpr int kSnapLds = 9216;        // floats of a conv tile in LDS (36 KB)
// Entry table over parameter vector [0, d): the given convs' weights (sorted
// by src, disjoint, channel counts multiples of the 16-byte vector width) as
// conv entries, everything else as copy entries, into out[0 .. *n_out)
// (at most 2 * n_convs + 1 entries; max_out is out's capacity).  Returns
// the number of workgroups, or -1 for an invalid list or too small an out;
// *bytes gets the algorithmic HBM bytes (4 read + 2 x element size written
// per conv weight, 8 per copied float).
long snapshot_table(const SnapConvDesc* convs, int n_convs, long d, int dt, SnapEntry* out, int max_out,
                    int* n_out, double* bytes);
hipError_t launch_snapshot(int dt, const float* x, float* v, const SnapEntry* tab_dev, int n_ent, long n_tiles,
                           void* wbase, hipStream_t st);
// The same snapshot with its work table in a fixed device array of
// kSnapScratchEntries entries (no allocation; lists of up to
// kSnapNoallocConvs convs).  Waits for the stream before returning.
// *bad_list = 1 (and nothing launched) for a list the table cannot take.
constexpr int kSnapNoallocConvs = 128;
constexpr int kSnapScratchEntries = 2 * kSnapNoallocConvs + 1;
hipError_t snapshot_noalloc(int dt, const SnapConvDesc* convs, int n_convs, long d, const float* x, float* v,
                            void* wbase, hipStream_t st, int* bad_list);

// Block update (Alg. 1 updater's last step), e in [lo, hi):
//   m = mu*m + g + wd*x; x -= lr*m   (m == null: x -= lr*(g + wd*x))
// (lr taken from args when args is not null)
hipError_t launch_sgd_update(float* x, float* m, const float* g, long lo, long hi, const StepArgs* args, float lr,
                             float mu, float wd, hipStream_t st);
// Averaging round (Alg. 1 averager) over n_rep replicas of n floats.
constexpr int kMaxReplicas = 16;
struct RepPtrs { float* p[kMaxReplicas]; };
hipError_t launch_average(const RepPtrs& reps, int n_rep, long n, hipStream_t st);

}  // namespace lpp
