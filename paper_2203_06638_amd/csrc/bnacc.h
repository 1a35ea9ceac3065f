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

#include "act.h"
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

// Per-channel moments of an MFMA output tile, for the batch sums of the
// producing conv's epilogue.  Each lane of wave (wm, wn) holds acc[x][y][i]:
// its TM x 4 rows (x, i), of which valid(x, i) lie inside the tensor, in
// column (wn TN + y) 16 + lane % 16.  A lane takes the count, mean and sum of
// squared deviations of its valid rows (two passes in registers); the lanes
// of a column are merged over the four lane groups (xor 16, then 32) and the
// WM row waves in order by the pairwise rule
//   n = na + nb,  mean = ma + (mb - ma) nb / n,  M2 = M2a + M2b + (mb - ma)^2 na nb / n,
// and out(t, n, mean, M2) runs for the tile's columns t < BN.  One barrier;
// red holds WM x 3 x BN floats of LDS.
// ALL: every row is valid, so merged counts are equal and known (no
// divisions); otherwise the weights use the hardware reciprocal (about one
// ulp, far below the statistics' use).
template <int TM, int TN, int WM, int BN, bool ALL, class Valid, class Out>
__device__ __forceinline__ void tile_moments(const f4 (&acc)[TM][TN], int wm, int wn, Valid valid,
                                             float (&red)[WM][3][BN], Out out) {
    const int lane = threadIdx.x & 63;
    float cl = 0.f;
#pragma unroll
    for (int x = 0; x < TM; ++x)
#pragma unroll
        for (int i = 0; i < 4; ++i) cl += (ALL || valid(x, i)) ? 1.f : 0.f;
#pragma unroll
    for (int y = 0; y < TN; ++y) {
        float cnt = cl, mu = 0.f, m2 = 0.f;
#pragma unroll
        for (int x = 0; x < TM; ++x)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                if (ALL || valid(x, i)) mu += acc[x][y][i];
        if (ALL) mu *= 1.f / (4 * TM);
        else mu = cnt > 0.f ? mu * __builtin_amdgcn_rcpf(cnt) : 0.f;
#pragma unroll
        for (int x = 0; x < TM; ++x)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float dv = acc[x][y][i] - mu;
                if (ALL || valid(x, i)) m2 += dv * dv;
            }
#pragma unroll
        for (int o = 16; o <= 32; o <<= 1) {
            const float co = __shfl_xor(cnt, o), mo = __shfl_xor(mu, o), qo = __shfl_xor(m2, o);
            const float n = cnt + co, d = mo - mu;
            if (ALL) {
                // equal counts: mean (a + b) / 2, M2 += d^2 n / 4
                m2 = (m2 + qo) + d * d * (0.25f * n);
                mu = 0.5f * (mu + mo);
            } else if (n > 0.f) {
                const float r = __builtin_amdgcn_rcpf(n);
                mu += d * (co * r);
                m2 += qo + d * d * (cnt * co * r);
            }
            cnt = n;
        }
        if (lane < 16) {
            const int col = (wn * TN + y) * 16 + lane;
            red[wm][0][col] = cnt;
            red[wm][1][col] = mu;
            red[wm][2][col] = m2;
        }
    }
    __syncthreads();
    const int t = threadIdx.x;
    if (t < BN) {
        float cnt = red[0][0][t], mu = red[0][1][t], m2 = red[0][2][t];
#pragma unroll
        for (int w = 1; w < WM; ++w) {
            const float cb = red[w][0][t], n = cnt + cb, d = red[w][1][t] - mu;
            if (ALL) {
                // counts w k and k: weights 1 / (w + 1) and w k / (w + 1)
                mu += d * (1.f / (w + 1));
                m2 += red[w][2][t] + d * d * (cb * ((float)w / (w + 1)));
            } else if (n > 0.f) {
                const float r = __builtin_amdgcn_rcpf(n);
                mu += d * (cb * r);
                m2 += red[w][2][t] + d * d * (cnt * cb * r);
            }
            cnt = n;
        }
        out(t, cnt, mu, m2);
    }
}

// A tile's moments into the batch sums: sum x = n mean and sum x^2 = M2 +
// n mean^2 added to the fp64 accumulators, or the tile's mean and M2 as the
// fixed-order partials of tile `tile`
__device__ __forceinline__ void tile_moments_store(const BnSums& sums, int tile, int C, int c, float n, float mu,
                                                   float m2) {
    if (sums.acc) {
        acc_add(sums.acc, 0, tile, C, c, (double)mu * n);
        acc_add(sums.acc, 1, tile, C, c, (double)m2 + (double)n * mu * mu);
    } else {
        sums.p0[(long)tile * C + c] = mu;
        sums.p1[(long)tile * C + c] = m2;
    }
}

}  // namespace lpp
