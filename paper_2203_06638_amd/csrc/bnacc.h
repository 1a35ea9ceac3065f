// bnacc.h -- batch-norm reductions merged across workgroups.
//
// The kernel that produces a reduced quantity (the conv epilogue for the
// forward batch sums, the backward reduce for sum g and sum g*xhat) adds each
// workgroup's fp64 partial into per-channel accumulators with device-scope
// atomics; the kernel that consumes them (batch-norm apply, backward apply)
// reads the accumulators in its prologue.  Adds are spread over kAccSlots
// copies (acc_add) to limit contention; readers sum the copies in a fixed
// order.  The accumulators are zeroed by the first
// kernel of every step.  fp64 addition order varies with workgroup timing, so
// the merged sums may differ run to run in their last fp64 bits (about
// 1e-16 relative), far below the fp32 values derived from them.
#pragma once
#include <hip/hip_runtime.h>

#include "kernels.h"

namespace lpp {

// Workgroup b adds to copy (b / 8) mod kAccSlots: the dispatcher deals
// consecutive workgroups to the eight XCDs in turn, so this spreads each
// XCD's workgroups over all copies (measured +0.4% on ResNet-20 against
// copy b mod kAccSlots, where all of an XCD's adds meet at one copy).
__device__ __forceinline__ void acc_add(double* acc, int q, int b, int C, int c, double v) {
    const int slot = (b >> 3) & (kAccSlots - 1);
    unsafeAtomicAdd(acc + ((long)q * kAccSlots + slot) * C + c, v);
}

__device__ __forceinline__ double acc_read(const double* acc, int q, int C, int c) {
    double s = 0.0;
#pragma unroll
    for (int k = 0; k < kAccSlots; ++k) s += acc[((long)q * kAccSlots + k) * C + c];
    return s;
}

// Scale and shift of a training-mode batch norm for channels c = threadIdx.x,
// threadIdx.x + blockDim.x, ... into sc / sh (LDS).  From the batch sums:
//   mean = S1 / M,  var = S2 / M - mean^2 (biased),  rstd = 1 / sqrt(var + eps),
//   scale = gamma * rstd,  shift = beta - mean * scale
// (fp64), and the first workgroup stores mean, rstd, scale, shift into aux;
// without acc, scale and shift are read from aux.
__device__ __forceinline__ void bn_fwd_coeffs(const BnFwd& b, int C, float* sc, float* sh) {
    for (int c = threadIdx.x; c < C; c += blockDim.x) {
        if (b.acc) {
            const double mu = acc_read(b.acc, 0, C, c) / (double)b.M;
            double var = acc_read(b.acc, 1, C, c) / (double)b.M - mu * mu;
            var = var > 0.0 ? var : 0.0;
            const double r = 1.0 / sqrt(var + (double)b.eps);
            const double s = (double)b.gamma[c] * r;
            const double t = (double)b.beta[c] - mu * s;
            sc[c] = (float)s;
            sh[c] = (float)t;
            if (blockIdx.x == 0 && b.aux) {
                b.aux[c] = (float)mu;
                b.aux[C + c] = (float)r;
                b.aux[2 * C + c] = (float)s;
                b.aux[3 * C + c] = (float)t;
            }
        } else {
            sc[c] = b.aux[2 * C + c];
            sh[c] = b.aux[3 * C + c];
        }
    }
}

}  // namespace lpp
