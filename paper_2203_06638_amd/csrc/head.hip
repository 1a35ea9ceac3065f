// head.hip -- the classifier head of the step: global average pool of the
// last feature map, the linear layer (the logits) and softmax cross-entropy
// against the step's labels, and their backward.
//
// Two forms, chosen per model by head_wide(C, O):
//  * fused (narrow heads, C x O small): one workgroup per sample pools its
//    features, forms its logits and its loss in one kernel;
//  * wide (C x O large, e.g. 2048 x 1000): pooling, then the logits as a
//    small matrix product on the matrix cores that reads the weight matrix
//    once, then a softmax kernel per sample; the input gradient likewise
//    (dz W on the matrix cores, then the broadcast over the pooled pixels).
// The weight matrix is row-major [O][C]; features are fp32 [N][C]; logits and
// dz are fp32 [N][O].  Every reduction runs in a fixed order.
#include "act.h"
#include "kernels.h"
#include "launch.h"

namespace lpp {

namespace {

inline unsigned nblk(long n, int per) { return (unsigned)((n + per - 1) / per); }

constexpr int kHeadMaxC = 2048, kHeadMaxO = 4096;
constexpr int kWaves = 8;    // waves per workgroup of the matrix-core kernels
constexpr int kTiles = 8;    // 16-row tiles of samples per workgroup

__device__ __forceinline__ f4 mfma4(float a, float b, f4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// Softmax cross-entropy of one sample whose O logits sit in LDS (z_s), 256
// threads: max and sum over classes as fixed-shape trees, then
// dz = (softmax - onehot(y)) / N and the sample's loss lse - z_y.
__device__ void softmax_ce_row(const float* z_s, int O, int y, int Nb, float* red, float* __restrict__ dz_row,
                               float* __restrict__ loss) {
    const int t = threadIdx.x;
    float mx = -INFINITY;
    for (int o = t; o < O; o += 256) mx = fmaxf(mx, z_s[o]);
    red[t] = mx;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if (t < w) red[t] = fmaxf(red[t], red[t + w]);
        __syncthreads();
    }
    const float zmax = red[0];
    __syncthreads();
    float se = 0.f;
    for (int o = t; o < O; o += 256) se += expf(z_s[o] - zmax);
    red[t] = se;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if (t < w) red[t] += red[t + w];
        __syncthreads();
    }
    const float lse = zmax + logf(red[0]);
    for (int o = t; o < O; o += 256) dz_row[o] = (expf(z_s[o] - lse) - (o == y ? 1.f : 0.f)) / (float)Nb;
    if (t == 0) *loss = lse - z_s[y];
}

// ---- fused form --------------------------------------------------------

// One workgroup per sample: pooled features f (also written out for the
// weight gradient), logits W f + b, softmax cross-entropy.  Pooling: thread
// (q, l) sums channel quad q over pixels l, l + rl, ...; the rl partial sums
// of a quad are added in LDS in a fixed order.  C % 4 == 0.
template <class T>
__global__ __launch_bounds__(256) void head_fwd_k(const T* __restrict__ x, int Nb, int HW, int C,
                                                  const float* __restrict__ W, const float* __restrict__ b, int O,
                                                  const StepArgs* __restrict__ args, float* __restrict__ feat,
                                                  float* __restrict__ logits, float* __restrict__ dz,
                                                  float* __restrict__ loss_per) {
    __shared__ __attribute__((aligned(16))) float f_s[kHeadMaxC];
    __shared__ float z_s[kHeadMaxO];
    __shared__ float red[256];
    __shared__ f4 part[256];
    const int n = blockIdx.x, t = threadIdx.x;
    const int C4 = C >> 2;
    for (int q0 = 0; q0 < C4; q0 += 256) {
        const int nq = min(256, C4 - q0), rl = 256 / nq;
        const int q = q0 + t % nq, l = t / nq;
        f4 s = f4{0.f, 0.f, 0.f, 0.f};
        if (l < rl)
            for (int e = l; e < HW; e += rl) s += ld4(x, ((long)n * HW + e) * C4 + q);
        part[t] = s;
        __syncthreads();
        if (t < nq) {
            f4 tot = part[t];
            for (int k = 1; k < rl; ++k) tot += part[k * nq + t];
            const f4 f = tot / (float)HW;
            *(f4*)(f_s + 4 * (q0 + t)) = f;
            *(f4*)(feat + (long)n * C + 4 * (q0 + t)) = f;
        }
        __syncthreads();
    }
    for (int o = t; o < O; o += 256) {
        float z = b ? b[o] : 0.f;
        const float* w = W + (long)o * C;
        for (int c = 0; c < C; ++c) z += w[c] * f_s[c];
        z_s[o] = z;
        logits[(long)n * O + o] = z;
    }
    __syncthreads();
    softmax_ce_row(z_s, O, args->labels[n], Nb, red, dz + (long)n * O, loss_per + n);
}

// one workgroup per sample: df = (dz W) / HW, broadcast over the HW pixels
template <class T>
__global__ __launch_bounds__(256) void head_bwd_x_k(const float* __restrict__ dz, const float* __restrict__ W,
                                                    int Nb, int HW, int C, int O, T* __restrict__ dx, int acc) {
    __shared__ float df[kHeadMaxC];
    const int n = blockIdx.x, t = threadIdx.x;
    for (int c = t; c < C; c += 256) {
        float s = 0.f;
        for (int o = 0; o < O; ++o) s += dz[(long)n * O + o] * W[(long)o * C + c];
        df[c] = s / (float)HW;
    }
    __syncthreads();
    const int C4 = C >> 2;
    T* out = dx + (long)n * HW * C;
    for (int i = t; i < HW * C4; i += 256) {
        const int c = (i % C4) * 4;
        const f4 v = f4{df[c], df[c + 1], df[c + 2], df[c + 3]};
        st4(out, i, acc ? ld4(out, i) + v : v);
    }
}

// ---- weight gradient (both forms) ----------------------------------------

// Narrow heads: one workgroup per class o.  dW[o][:] = sum_n dz[n][o] f[n][:]
// with thread (q, l) summing channel quad q over samples l, l + rl, ... and the
// partial sums added in LDS in a fixed order; db[o] likewise.  Workgroup 0
// also forms the batch-mean loss.  C % 4 == 0.
__global__ __launch_bounds__(256) void head_bwd_w_rows_k(const float* __restrict__ dz, const float* __restrict__ feat,
                                                         int Nb, int C, int O, float* __restrict__ gW,
                                                         float* __restrict__ gb, const float* __restrict__ loss_per,
                                                         float* __restrict__ loss) {
    __shared__ f4 part[256];
    __shared__ float pb[256];
    const int o = blockIdx.x, t = threadIdx.x;
    if (o == 0 && t == 0) {
        float s = 0.f;
        for (int n = 0; n < Nb; ++n) s += loss_per[n];
        loss[0] = s / (float)Nb;
    }
    if (!gW) return;
    const int C4 = C >> 2;
    for (int q0 = 0; q0 < C4; q0 += 256) {
        const int nq = min(256, C4 - q0), rl = 256 / nq;
        const int q = q0 + t % nq, l = t / nq;
        f4 s = f4{0.f, 0.f, 0.f, 0.f};
        if (l < rl)
            for (int n = l; n < Nb; n += rl) s += dz[(long)n * O + o] * ld4(feat, (long)n * C4 + q);
        part[t] = s;
        __syncthreads();
        if (t < nq) {
            f4 tot = part[t];
            for (int k = 1; k < rl; ++k) tot += part[k * nq + t];
            float* g = gW + (long)o * C + 4 * (q0 + t);   // any alignment: scalar stores
            g[0] = tot[0];
            g[1] = tot[1];
            g[2] = tot[2];
            g[3] = tot[3];
        }
        __syncthreads();
    }
    if (gb) {
        float s = 0.f;
        for (int n = t; n < Nb; n += 256) s += dz[(long)n * O + o];
        pb[t] = s;
        __syncthreads();
        for (int w = 128; w > 0; w >>= 1) {
            if (t < w) pb[t] += pb[t + w];
            __syncthreads();
        }
        if (t == 0) gb[o] = pb[0];
    }
}

// dW[o][c] = sum_n dz[n][o] f[n][c], db[o] = sum_n dz[n][o], samples in
// order; thread 0 of block 0 also forms the batch-mean loss.  Q channels per
// thread (4 when C % 4 == 0).
template <int Q>
__global__ void head_bwd_w_k(const float* __restrict__ dz, const float* __restrict__ feat, int Nb, int C, int O,
                             float* __restrict__ gW, float* __restrict__ gb, const float* __restrict__ loss_per,
                             float* __restrict__ loss) {
    const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx == 0) {
        float s = 0.f;
        for (int n = 0; n < Nb; ++n) s += loss_per[n];
        loss[0] = s / (float)Nb;
    }
    if (!gW) return;
    const int CQ = C / Q;
    if (idx < (long)O * CQ) {
        const int o = (int)(idx / CQ), c = (int)(idx - (long)o * CQ) * Q;
        float s[Q];
#pragma unroll
        for (int k = 0; k < Q; ++k) s[k] = 0.f;
        for (int n = 0; n < Nb; ++n) {
            const float d = dz[(long)n * O + o];
            const float* fr = feat + (long)n * C + c;
#pragma unroll
            for (int k = 0; k < Q; ++k) s[k] += d * fr[k];
        }
#pragma unroll
        for (int k = 0; k < Q; ++k) gW[(long)o * C + c + k] = s[k];
    } else if (gb && idx < (long)O * CQ + O) {
        const int o = (int)(idx - (long)O * CQ);
        float s = 0.f;
        for (int n = 0; n < Nb; ++n) s += dz[(long)n * O + o];
        gb[o] = s;
    }
}

// ---- wide form -----------------------------------------------------------
//
// Matrix-core mapping (v_mfma_f32_16x16x4_f32): A is 16 x 4, B is 4 x 16,
// lane l supplies A[l%16][l/16] and B[l/16][l%16]; lane l holds
// D[4*(l/16)+v][l%16], v = 0..3.  The contraction index is permuted the same
// way on both operands: in contraction block kb (16 indices), lane l supplies
// index 16*kb + 4*(l/16) + j to step j of A and of B, so four steps sum
// exactly the block's 16 indices.  A workgroup's waves take the blocks
// round-robin and their partial tiles are added in wave order in LDS.

// z[n][o] = b[o] + sum_c W[o][c] f[n][c]: one workgroup per 16 outputs (rows
// of D) and up to kTiles tiles of 16 samples (columns of D).  C % 16 == 0.
__global__ __launch_bounds__(512) void head_logits_k(const float* __restrict__ W, const float* __restrict__ b,
                                                     const float* __restrict__ f, float* __restrict__ z, int Nb,
                                                     int C, int O) {
    __shared__ float part[kWaves][kTiles][256];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int r = lane & 15, g = lane >> 4;
    const int o0 = blockIdx.x * 16, t0 = blockIdx.y * kTiles;
    const int nt = min(kTiles, (Nb + 15) / 16 - t0);
    const bool ov = o0 + r < O;
    const float* wrow = W + (long)(ov ? o0 + r : 0) * C + 4 * g;
    f4 acc[kTiles];
#pragma unroll
    for (int t = 0; t < kTiles; ++t) acc[t] = f4{0.f, 0.f, 0.f, 0.f};
    for (int kb = wv; kb < C / 16; kb += kWaves) {
        const f4 a = ov ? *(const f4*)(wrow + 16 * kb) : f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int t = 0; t < kTiles; ++t) {
            if (t < nt) {
                const int n = (t0 + t) * 16 + r;
                const f4 bv = n < Nb ? *(const f4*)(f + (long)n * C + 16 * kb + 4 * g) : f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[t] = mfma4(a[j], bv[j], acc[t]);
            }
        }
    }
#pragma unroll
    for (int t = 0; t < kTiles; ++t)
        if (t < nt)
#pragma unroll
            for (int v = 0; v < 4; ++v) part[wv][t][v * 64 + lane] = acc[t][v];
    __syncthreads();
    for (int e = threadIdx.x; e < nt * 256; e += 512) {
        const int t = e >> 8, q = e & 255;
        float s = 0.f;
        for (int w = 0; w < kWaves; ++w) s += part[w][t][q];
        const int v = q >> 6, ln = q & 63;
        const int o = o0 + 4 * (ln >> 4) + v, n = (t0 + t) * 16 + (ln & 15);
        if (o < O && n < Nb) z[(long)n * O + o] = (b ? b[o] : 0.f) + s;
    }
}

// One workgroup per sample: softmax cross-entropy of its logits row.
__global__ __launch_bounds__(256) void head_softmax_k(const float* __restrict__ z, int Nb, int O,
                                                      const StepArgs* __restrict__ args, float* __restrict__ dz,
                                                      float* __restrict__ loss_per) {
    __shared__ float z_s[kHeadMaxO];
    __shared__ float red[256];
    const int n = blockIdx.x;
    for (int o = threadIdx.x; o < O; o += 256) z_s[o] = z[(long)n * O + o];
    __syncthreads();
    softmax_ce_row(z_s, O, args->labels[n], Nb, red, dz + (long)n * O, loss_per + n);
}

// df[n][c] = sum_o dz[n][o] W[o][c]: one workgroup per 16 channels (rows of
// D, A = W transposed) and up to kTiles tiles of 16 samples (columns of D,
// B = dz transposed); the contraction runs over the O classes, zero-padded
// to a multiple of 16.
__global__ __launch_bounds__(512) void head_dfeat_k(const float* __restrict__ dz, const float* __restrict__ W,
                                                    float* __restrict__ df, int Nb, int C, int O) {
    __shared__ float part[kWaves][kTiles][256];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int r = lane & 15, g = lane >> 4;
    const int c0 = blockIdx.x * 16, t0 = blockIdx.y * kTiles;
    const int nt = min(kTiles, (Nb + 15) / 16 - t0);
    f4 acc[kTiles];
#pragma unroll
    for (int t = 0; t < kTiles; ++t) acc[t] = f4{0.f, 0.f, 0.f, 0.f};
    for (int kb = wv; kb < (O + 15) / 16; kb += kWaves) {
        const int o = 16 * kb + 4 * g;
        f4 a;
#pragma unroll
        for (int j = 0; j < 4; ++j) a[j] = o + j < O ? W[(long)(o + j) * C + c0 + r] : 0.f;
#pragma unroll
        for (int t = 0; t < kTiles; ++t) {
            if (t < nt) {
                const int n = (t0 + t) * 16 + r;
                f4 bv = f4{0.f, 0.f, 0.f, 0.f};
                if (n < Nb) {
                    const float* zr = dz + (long)n * O + o;
#pragma unroll
                    for (int j = 0; j < 4; ++j) bv[j] = o + j < O ? zr[j] : 0.f;
                }
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[t] = mfma4(a[j], bv[j], acc[t]);
            }
        }
    }
#pragma unroll
    for (int t = 0; t < kTiles; ++t)
        if (t < nt)
#pragma unroll
            for (int v = 0; v < 4; ++v) part[wv][t][v * 64 + lane] = acc[t][v];
    __syncthreads();
    for (int e = threadIdx.x; e < nt * 256; e += 512) {
        const int t = e >> 8, q = e & 255;
        float s = 0.f;
        for (int w = 0; w < kWaves; ++w) s += part[w][t][q];
        const int v = q >> 6, ln = q & 63;
        const int c = c0 + 4 * (ln >> 4) + v, n = (t0 + t) * 16 + (ln & 15);
        if (n < Nb) df[(long)n * C + c] = s;
    }
}

}  // namespace

bool head_wide(int C, int O) { return C % 16 == 0 && (long)C * O >= kHeadWideMin; }

hipError_t launch_head_fwd(int dt, const void* x, int Nb, int HW, int C, const float* W, const float* b, int O,
                           const StepArgs* args, float* feat, float* logits, float* dz, float* loss_per,
                           hipStream_t st) {
    if (O > kHeadMaxO) return hipErrorInvalidValue;
    if (head_wide(C, O)) {
        hipError_t e = launch_gap_fwd(dt, x, feat, Nb, HW, C, st);
        if (e != hipSuccess) return e;
        const dim3 grid(nblk(O, 16), nblk(Nb, 16 * kTiles));
        launch(head_logits_k, grid, dim3(64 * kWaves), 0, st, W, b, (const float*)feat, logits, Nb, C, O);
        launch(head_softmax_k, dim3(Nb), dim3(256), 0, st, (const float*)logits, Nb, O, args, dz, loss_per);
        return hipGetLastError();
    }
    if (C > kHeadMaxC) return hipErrorInvalidValue;
    if (dt == DT_BF16)
        launch(head_fwd_k<bf16>, dim3(Nb), dim3(256), 0, st, (const bf16*)x, Nb, HW, C, W, b, O, args, feat, logits,
               dz, loss_per);
    else
        launch(head_fwd_k<float>, dim3(Nb), dim3(256), 0, st, (const float*)x, Nb, HW, C, W, b, O, args, feat,
               logits, dz, loss_per);
    return hipGetLastError();
}

hipError_t launch_head_bwd_w(const float* dz, const float* feat, int Nb, int C, int O, float* gW, float* gb,
                             const float* loss_per, float* loss, hipStream_t st) {
    if (gW && C % 4 == 0 && !head_wide(C, O)) {
        launch(head_bwd_w_rows_k, dim3(O), dim3(256), 0, st, dz, feat, Nb, C, O, gW, gb, loss_per, loss);
    } else if (gW && C % 4 == 0) {
        const long n = (long)O * (C / 4) + O;
        launch(head_bwd_w_k<4>, dim3(nblk(n, 256)), dim3(256), 0, st, dz, feat, Nb, C, O, gW, gb, loss_per, loss);
    } else {
        const long n = gW ? (long)O * C + O : 1;
        launch(head_bwd_w_k<1>, dim3(nblk(n, 256)), dim3(256), 0, st, dz, feat, Nb, C, O, gW, gb, loss_per, loss);
    }
    return hipGetLastError();
}

hipError_t launch_head_bwd_x(int dt, const float* dz, const float* W, int Nb, int HW, int C, int O, void* dx,
                             bool acc, float* scratch, hipStream_t st) {
    if (head_wide(C, O)) {
        if (!scratch) return hipErrorInvalidValue;
        const dim3 grid(C / 16, nblk(Nb, 16 * kTiles));
        launch(head_dfeat_k, grid, dim3(64 * kWaves), 0, st, dz, W, scratch, Nb, C, O);
        return launch_gap_bwd(dt, scratch, dx, Nb, HW, C, acc, st);
    }
    if (C > kHeadMaxC) return hipErrorInvalidValue;
    if (dt == DT_BF16)
        launch(head_bwd_x_k<bf16>, dim3(Nb), dim3(256), 0, st, dz, W, Nb, HW, C, O, (bf16*)dx, (int)acc);
    else
        launch(head_bwd_x_k<float>, dim3(Nb), dim3(256), 0, st, dz, W, Nb, HW, C, O, (float*)dx, (int)acc);
    return hipGetLastError();
}

}  // namespace lpp
