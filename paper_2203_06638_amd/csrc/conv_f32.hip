// conv_f32.hip -- fp32 convolution passes on gfx950 matrix cores.
//
// Forward and data-gradient passes are one implicit GEMM
//     Y[m][n] = sum_k A[m][k] * B[n][k]
// with m an output pixel (NHWC), n an output channel, and k = (r, s, c) a
// filter tap and source channel.  A is gathered on the fly from the NHWC
// source activation; B is a weight matrix whose rows are contiguous in k
// (the snapshot writes both the forward layout W_f[cout][r][s][cin] and the
// data-gradient layout W_d[cin][r][s][cout]).
//
// Matrix-core mapping (v_mfma_f32_16x16x4_f32, 64 lanes): lane l supplies
// A[row = l%16][k = l/16] and B[k = l/16][col = l%16] and holds
// D[4*(l/16) + i][l%16], i = 0..3.  Each lane loads a float4 of four
// consecutive channels for its row (pixel) and its column (filter row); the
// four components feed four successive MFMAs, so the 16 k-values a lane
// group covers per float4 are permuted identically in A and B (the sum is
// over all of them either way).
//
// Weight gradient: dW[cout][(r,s,c)] = sum over output pixels p of
// dY[p][cout] * X_im2col[p][(r,s,c)] -- a GEMM whose reduction runs over
// N*Ho*Wo pixels.  Pixel chunks of 64 are staged through LDS (dY rows and
// im2col rows as loaded, float4 along channels); each wave reduces 16 of the
// chunk's pixels; waves are summed in a fixed order and every split of the
// pixel range writes its own partial, summed in order by a second kernel.
// Convolution outputs and weight gradients use no atomics and are bitwise
// reproducible; only the batch-norm sums of the forward epilogue are merged
// across workgroups by fp64 atomic adds (bnacc.h).
#include <algorithm>
#include <cstdint>

#include "bnacc.h"
#include "kernels.h"
#include "launch.h"

namespace lpp {

typedef float f4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f4 relu4(f4 v) {
    return f4{fmaxf(v[0], 0.f), fmaxf(v[1], 0.f), fmaxf(v[2], 0.f), fmaxf(v[3], 0.f)};
}

__device__ __forceinline__ f4 mfma16x16x4(float a, float b, f4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// Copies n float4 into LDS: addr(i, src, dst) names element i's source (null:
// zero) and LDS destination.  Each thread issues NB global loads before their
// LDS stores, so the load latencies overlap instead of adding up.
template <int NB, class Addr>
__device__ __forceinline__ void lds_stage(int n, Addr addr) {
    for (int base = threadIdx.x; base < n; base += NB * 256) {
        f4 v[NB];
        float* d[NB];
#pragma unroll
        for (int u = 0; u < NB; ++u) {
            const int i = base + u * 256;
            const float* src = nullptr;
            d[u] = nullptr;
            if (i < n) addr(i, src, d[u]);
            v[u] = src ? *(const f4*)src : f4{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
        for (int u = 0; u < NB; ++u)
            if (d[u]) *(f4*)d[u] = v[u];
    }
}

// Offset of source pixel (n, hs, ws) feeding output pixel (n, p, q) through
// tap (r, s), or -1 when the tap falls in the zero padding / between strides.
template <int MODE>
__device__ __forceinline__ int src_pixel(int n, int p, int q, int r, int s, const ConvGeom& g) {
    int hs, ws;
    if (MODE == CONV_FWD) {
        hs = p * g.stride - g.pad + r;
        ws = q * g.stride - g.pad + s;
    } else {
        // dX[p][q] gathers dY[(p + pad - r)/stride][(q + pad - s)/stride]
        int hn = p + g.pad - r, wn = q + g.pad - s;
        if (hn < 0 || wn < 0) return -1;
        if (g.stride != 1) {
            if ((hn % g.stride) | (wn % g.stride)) return -1;
            hn /= g.stride;
            wn /= g.stride;
        }
        hs = hn;
        ws = wn;
    }
    if (hs < 0 || hs >= g.Hs || ws < 0 || ws >= g.Ws) return -1;
    return ((n * g.Hs + hs) * g.Ws + ws) * g.Cs;
}

// WM waves along m (4/WM along n); each wave owns TM x TN tiles of 16x16.
// FAST: Cs % 16 == 0, so a group of four float4 chunks never straddles a tap.
// STATS: also form, per output channel, the mean and the sum of squared
// deviations over this workgroup's BM output rows and add the tile's share of
// the batch sums (sum y, sum y^2) into the batch-norm accumulators.
template <int MODE, int WM, int TM, int TN, bool FAST, bool STATS>
__global__ __launch_bounds__(256) void conv_igemm_f32(const float* __restrict__ src, const float* __restrict__ B,
                                                      const float* __restrict__ bias, float* __restrict__ Y,
                                                      ConvGeom g, int accumulate, BnSums sums) {
    constexpr int WN = 4 / WM;
    constexpr int BM = WM * TM * 16, BN = WN * TN * 16;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wm = wave % WM, wn = wave / WM;
    const int gi = lane >> 4, li = lane & 15;
    const int HoWo = g.Ho * g.Wo;
    const int M = g.Nb * HoWo;
    const int Ktot = g.R * g.S * g.Cs;
    const int m_base = blockIdx.x * BM + wm * TM * 16;
    const int n_base = blockIdx.y * BN + wn * TN * 16;

    int an[TM], ap[TM], aq[TM];
    bool av[TM];
#pragma unroll
    for (int t = 0; t < TM; ++t) {
        int m = m_base + t * 16 + li;
        av[t] = m < M;
        int mm = av[t] ? m : 0;
        an[t] = mm / HoWo;
        int rem = mm - an[t] * HoWo;
        ap[t] = rem / g.Wo;
        aq[t] = rem - ap[t] * g.Wo;
    }
    const float* bp[TN];
    bool bv[TN];
#pragma unroll
    for (int t = 0; t < TN; ++t) {
        int n = n_base + t * 16 + li;
        bv[t] = n < g.Ncols;
        bp[t] = B + (long)(bv[t] ? n : 0) * Ktot;
    }
    f4 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};

    if (FAST) {
        for (int r = 0; r < g.R; ++r)
            for (int s = 0; s < g.S; ++s) {
                int so[TM];
#pragma unroll
                for (int t = 0; t < TM; ++t) so[t] = av[t] ? src_pixel<MODE>(an[t], ap[t], aq[t], r, s, g) : -1;
                const int kt = (r * g.S + s) * g.Cs;
                for (int c0 = 4 * gi; c0 < g.Cs; c0 += 16) {
                    f4 a[TM], b[TN];
#pragma unroll
                    for (int t = 0; t < TM; ++t)
                        a[t] = so[t] >= 0 ? *(const f4*)(src + so[t] + c0) : f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int t = 0; t < TN; ++t)
                        b[t] = bv[t] ? *(const f4*)(bp[t] + kt + c0) : f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int j = 0; j < 4; ++j)
#pragma unroll
                        for (int x = 0; x < TM; ++x)
#pragma unroll
                            for (int y = 0; y < TN; ++y) acc[x][y] = mfma16x16x4(a[x][j], b[y][j], acc[x][y]);
                }
            }
    } else {
        const int Cq = g.Cs >> 2;   // float4 chunks per tap
        const int KC = Ktot >> 2;   // float4 chunks in all of k
        for (int kc0 = 0; kc0 < KC; kc0 += 4) {
            const int kc = kc0 + gi;
            f4 a[TM], b[TN];
#pragma unroll
            for (int t = 0; t < TM; ++t) a[t] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int t = 0; t < TN; ++t) b[t] = f4{0.f, 0.f, 0.f, 0.f};
            if (kc < KC) {
                int tap = kc / Cq;
                int c = (kc - tap * Cq) * 4;
                int r = tap / g.S, s = tap - r * g.S;
#pragma unroll
                for (int t = 0; t < TM; ++t) {
                    int so = av[t] ? src_pixel<MODE>(an[t], ap[t], aq[t], r, s, g) : -1;
                    if (so >= 0) a[t] = *(const f4*)(src + so + c);
                }
#pragma unroll
                for (int t = 0; t < TN; ++t)
                    if (bv[t]) b[t] = *(const f4*)(bp[t] + kc * 4);
            }
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int x = 0; x < TM; ++x)
#pragma unroll
                    for (int y = 0; y < TN; ++y) acc[x][y] = mfma16x16x4(a[x][j], b[y][j], acc[x][y]);
        }
    }

#pragma unroll
    for (int y = 0; y < TN; ++y) {
        const int n = n_base + y * 16 + li;
        const float bb = (bias && n < g.Ncols) ? bias[n] : 0.f;
#pragma unroll
        for (int x = 0; x < TM; ++x)
#pragma unroll
            for (int i = 0; i < 4; ++i) acc[x][y][i] += bb;
        if (n >= g.Ncols) continue;
#pragma unroll
        for (int x = 0; x < TM; ++x)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int m = m_base + x * 16 + gi * 4 + i;
                if (m >= M) continue;
                const long o = (long)m * g.Ncols + n;
                const float v = acc[x][y][i];
                Y[o] = accumulate == kStoreAdd ? Y[o] + v : (accumulate == kStoreRelu ? fmaxf(v, 0.f) : v);
            }
    }
    if (STATS) {
        __shared__ float red[WM][3][BN];
        const auto valid = [&](int x, int i) { return m_base + x * 16 + gi * 4 + i < M; };
        const auto store = [&](int t, float n, float mu, float m2) {
            if (blockIdx.y * BN + t < g.Ncols)
                tile_moments_store(sums, (int)blockIdx.x, g.Ncols, blockIdx.y * BN + t, n, mu, m2);
        };
        if ((int)blockIdx.x * BM + BM <= M) tile_moments<TM, TN, WM, BN, true>(acc, wm, wn, valid, red, store);
        else tile_moments<TM, TN, WM, BN, false>(acc, wm, wn, valid, red, store);
    }
}

// LDS-staged variant for Cs % 16 == 0.  A k-step is one filter tap and 16
// source channels.  The workgroup's A tile (BM rows x 16) and B tile (BN rows
// x 16) are loaded cooperatively as float4 (each thread keeps the same rows in
// every k-step, so row decoding happens once), double-buffered in LDS with the
// next k-step's global loads in flight during this k-step's MFMAs; one
// barrier per k-step.  Waves form a WM x WN grid over the tile; a wave owns
// TM x TN 16x16 output tiles and reads its operands as float4 from LDS.
template <int MODE, int BM, int BN, int WM, bool STATS>
__global__ __launch_bounds__(256) void conv_lds_f32(const float* __restrict__ src, const float* __restrict__ B,
                                                    const float* __restrict__ bias, float* __restrict__ Y,
                                                    ConvGeom g, int accumulate, BnSums sums) {
    constexpr int WN = 4 / WM;
    constexpr int TM = BM / (WM * 16), TN = BN / (WN * 16);
    constexpr int LDW = 20;                                  // 16 floats + 4 pad per LDS row
    constexpr int NA = (BM * 4 + 255) / 256, NB = (BN * 4 + 255) / 256;
    __shared__ float As[2][BM][LDW];
    __shared__ float Bs[2][BN][LDW];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave % WM, wn = wave / WM;
    const int gi = lane >> 4, li = lane & 15;
    const int HoWo = g.Ho * g.Wo;
    const int M = g.Nb * HoWo;
    const int Ktot = g.R * g.S * g.Cs;
    const int CG = g.Cs >> 4;                                // 16-channel groups per tap
    const int KS = g.R * g.S * CG;                           // k-steps
    const int m0 = blockIdx.x * BM, n0 = blockIdx.y * BN;
    const int quad = tid & 3;                                // each thread's float4 within a 16-wide row

    // rows of A this thread loads: (tid + 256 i) / 4
    int an[NA], ap[NA], aq[NA];
    bool av[NA];
#pragma unroll
    for (int i = 0; i < NA; ++i) {
        const int row = (tid + 256 * i) >> 2;
        const int m = m0 + row;
        av[i] = (tid + 256 * i) < BM * 4 && m < M;
        const int mm = av[i] ? m : 0;
        an[i] = mm / HoWo;
        const int rem = mm - an[i] * HoWo;
        ap[i] = rem / g.Wo;
        aq[i] = rem - ap[i] * g.Wo;
    }
    const float* brow[NB];
    bool bvld[NB];
#pragma unroll
    for (int i = 0; i < NB; ++i) {
        const int row = (tid + 256 * i) >> 2;
        const int n = n0 + row;
        bvld[i] = (tid + 256 * i) < BN * 4 && n < g.Ncols;
        brow[i] = B + (long)(bvld[i] ? n : 0) * Ktot + quad * 4;
    }

    f4 ra[NA], rb[NB];
    auto gload = [&](int ks) {
        const int tap = ks / CG;
        const int cg = ks - tap * CG;
        const int r = tap / g.S, sx = tap - r * g.S;
        const int c = cg * 16 + quad * 4;
#pragma unroll
        for (int i = 0; i < NA; ++i) {
            const int so = av[i] ? src_pixel<MODE>(an[i], ap[i], aq[i], r, sx, g) : -1;
            ra[i] = so >= 0 ? *(const f4*)(src + so + c) : f4{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
        for (int i = 0; i < NB; ++i) rb[i] = bvld[i] ? *(const f4*)(brow[i] + ks * 16) : f4{0.f, 0.f, 0.f, 0.f};
    };
    auto lstore = [&](int buf) {
#pragma unroll
        for (int i = 0; i < NA; ++i)
            if ((tid + 256 * i) < BM * 4) *(f4*)&As[buf][(tid + 256 * i) >> 2][quad * 4] = ra[i];
#pragma unroll
        for (int i = 0; i < NB; ++i)
            if ((tid + 256 * i) < BN * 4) *(f4*)&Bs[buf][(tid + 256 * i) >> 2][quad * 4] = rb[i];
    };

    f4 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};

    gload(0);
    lstore(0);
    __syncthreads();
    for (int ks = 0; ks < KS; ++ks) {
        const int buf = ks & 1;
        if (ks + 1 < KS) gload(ks + 1);
        f4 a[TM], b[TN];
#pragma unroll
        for (int x = 0; x < TM; ++x) a[x] = *(const f4*)&As[buf][(wm * TM + x) * 16 + li][gi * 4];
#pragma unroll
        for (int y = 0; y < TN; ++y) b[y] = *(const f4*)&Bs[buf][(wn * TN + y) * 16 + li][gi * 4];
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int x = 0; x < TM; ++x)
#pragma unroll
                for (int y = 0; y < TN; ++y) acc[x][y] = mfma16x16x4(a[x][j], b[y][j], acc[x][y]);
        if (ks + 1 < KS) lstore(buf ^ 1);
        __syncthreads();
    }

    const int m_base = m0 + wm * TM * 16;
    const int n_base = n0 + wn * TN * 16;
#pragma unroll
    for (int y = 0; y < TN; ++y) {
        const int n = n_base + y * 16 + li;
        const float bb = (bias && n < g.Ncols) ? bias[n] : 0.f;
#pragma unroll
        for (int x = 0; x < TM; ++x)
#pragma unroll
            for (int i = 0; i < 4; ++i) acc[x][y][i] += bb;
        if (n >= g.Ncols) continue;
#pragma unroll
        for (int x = 0; x < TM; ++x)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int m = m_base + x * 16 + gi * 4 + i;
                if (m >= M) continue;
                const long o = (long)m * g.Ncols + n;
                const float v = acc[x][y][i];
                Y[o] = accumulate == kStoreAdd ? Y[o] + v : (accumulate == kStoreRelu ? fmaxf(v, 0.f) : v);
            }
    }
    if (STATS) {
        __shared__ float red[WM][3][BN];
        const auto valid = [&](int x, int i) { return m_base + x * 16 + gi * 4 + i < M; };
        const auto store = [&](int t, float n, float mu, float m2) {
            if (n0 + t < g.Ncols) tile_moments_store(sums, (int)blockIdx.x, g.Ncols, n0 + t, n, mu, m2);
        };
        if (m0 + BM <= M) tile_moments<TM, TN, WM, BN, true>(acc, wm, wn, valid, red, store);
        else tile_moments<TM, TN, WM, BN, false>(acc, wm, wn, valid, red, store);
    }
}

template <int MODE, int BM, int BN, int WM>
static hipError_t launch_lds(const float* src, const float* B, const float* bias, float* Y, const ConvGeom& g,
                             int acc, const BnSums* stats, hipStream_t st) {
    const long M = (long)g.Nb * g.Ho * g.Wo;
    dim3 grid((unsigned)((M + BM - 1) / BM), (unsigned)((g.Ncols + BN - 1) / BN));
    if (stats)
        launch((conv_lds_f32<MODE, BM, BN, WM, true>), grid, dim3(256), 0, st, src, B, bias, Y, g,
                           (int)acc, stats ? *stats : BnSums{});
    else
        launch((conv_lds_f32<MODE, BM, BN, WM, false>), grid, dim3(256), 0, st, src, B, bias, Y, g,
                           (int)acc, stats ? *stats : BnSums{});
    return hipGetLastError();
}

// Spatially tiled variant (stride-1 data gradients and any forward pass with
// Cs % 16 == 0 whose tile shape fits): a workgroup computes OH full output
// rows of one image (TP = OH * Wo pixels) for BN output channels.  For each
// group of 16 source channels it loads the input rows the tile reads, halo
// and padding included (IH x IW pixels), and the filter slice (BN x R*S x
// 16) into LDS once, then runs every tap from LDS: the 3x3 halo is fetched
// from memory once instead of once per tap.  The data gradient of a stride-1
// conv is a forward conv of dY with the filter flipped and padding R-1-pad.
// IW_inv = ceil(2^32 / IW): pix / IW == umulhi(pix, IW_inv) for the pixel
// counts of an LDS tile (pix * IW < 2^32).
struct TileGeom { int OH, IH, IW, pad_eff, tiles_per_img; unsigned IW_inv; };

// INBN (forward passes): the source is the input of a training-mode batch
// norm followed by a ReLU; each staged source value becomes
// relu(fma(x, scale[c], shift[c])) (padding stays zero), with the per-channel
// coefficients derived in the prologue from the batch sums (or read from aux;
// bnacc.h).  The normalised tensor is never stored.
// Variants with at most two row blocks per wave and no epilogue statistics
// or folded input fit 128 registers without spilling: they are held to that,
// for four waves per SIMD instead of three.
// 16 bytes of device memory at p, through a global-address-space pointer (a
// pointer chosen at run time between buffers would otherwise be a flat
// address, whose loads also count with the LDS accesses)
__device__ __forceinline__ f4 ld_global4(const float* p) {
    return *(const __attribute__((address_space(1))) f4*)p;
}

template <int MODE, int KS, int WM, int TM, int TN, bool STATS, bool INBN>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu((TM <= 2 && !INBN && !STATS) ? 4 : 1, 8)))
void conv_tile_f32(const float* __restrict__ src, const float* __restrict__ B,
                                                     const float* __restrict__ bias, float* __restrict__ Y,
                                                     ConvGeom g, TileGeom t, int accumulate, BnSums sums, BnFwd inbn,
                                                     BnBwdSum bs) {
    constexpr int WN = 4 / WM;
    constexpr int TP = WM * TM * 16, BN = WN * TN * 16;
    constexpr int LDW = 20;
    constexpr int RS = KS * KS;
    constexpr int NU = 8;                         // float4 loads in flight per thread
    extern __shared__ float lds[];
    float* Xs = lds;                              // [IH*IW][LDW]
    float* Ws = lds + t.IH * t.IW * LDW;          // [BN*RS][LDW]
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave % WM, wn = wave / WM;
    const int gi = lane >> 4, li = lane & 15;
    const int img = blockIdx.x / t.tiles_per_img;
    const int oh0 = (blockIdx.x - img * t.tiles_per_img) * t.OH;
    const int n0 = blockIdx.y * BN;
    const int st = g.stride;
    const int h_org = oh0 * st - t.pad_eff, w_org = -t.pad_eff;
    const int npix = t.OH * g.Wo;

    __shared__ float in_co[INBN ? 2 * kFoldMaxC : 1];   // scale | shift of the source channels
    if (INBN) {
        bn_fwd_coeffs(inbn, g.Cs, in_co, in_co + kFoldMaxC);
        __syncthreads();
    }
    // relu(fma(v, scale, shift)) of source quad c..c+3 (INBN)
    auto fold = [&](f4 v, int c) {
        if (INBN) {
#pragma unroll
            for (int k = 0; k < 4; ++k) v[k] = fmaxf(__builtin_fmaf(v[k], in_co[c + k], in_co[kFoldMaxC + c + k]), 0.f);
        }
        return v;
    };

    // LDS offset of the input pixel each of this lane's output rows reads at tap (0,0)
    int abase[TM];
#pragma unroll
    for (int x = 0; x < TM; ++x) {
        int p = (wm * TM + x) * 16 + li;
        p = p < npix ? p : npix - 1;
        const int oh = p / g.Wo, ow = p - (p / g.Wo) * g.Wo;
        abase[x] = (oh * st * t.IW + ow * st) * LDW + gi * 4;
    }

    f4 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};

    // loader: element e = tid + 256 u has quad q = tid & 3 in both parts.
    // When a channel group fits one batch (ntot <= NU*256), the addresses
    // are decoded once and the next group's loads -- the same addresses 16
    // channels on -- are issued before this group's MFMAs.
    const int q = tid & 3;
    const int nx = t.IH * t.IW * 4, ntot = nx + BN * RS * 4;
    const int ngroups = g.Cs >> 4;
    // decode: the element's source quad sp (nullptr: none -- zero padding, a
    // column past the output) and its LDS offset d (-1: past the tiles)
    auto decode = [&](int e, const float*& sp, int& d) {
        sp = nullptr;
        d = -1;
        if (e < nx) {
            const int pix = e >> 2;
            const int ih = (int)__umulhi((unsigned)pix, t.IW_inv);
            const int iw = pix - ih * t.IW;
            const int h = h_org + ih, w = w_org + iw;
            if (h >= 0 && h < g.Hs && w >= 0 && w < g.Ws)
                sp = src + ((long)(img * g.Hs + h) * g.Ws + w) * g.Cs + q * 4;
            d = pix * LDW + q * 4;
        } else if (e < ntot) {
            const int rest = (e - nx) >> 2;
            const int tap = rest % RS, nl = rest / RS;
            const int n = n0 + nl;
            const int stap = MODE == CONV_FWD ? tap : RS - 1 - tap;
            if (n < g.Ncols) sp = B + ((long)n * RS + stap) * g.Cs + q * 4;
            d = t.IH * t.IW * LDW + rest * LDW + q * 4;
        }
    };
    auto compute = [&]() {
#pragma unroll
        for (int tap = 0; tap < RS; ++tap) {
            const int toff = ((tap / KS) * t.IW + tap % KS) * LDW;
            f4 a[TM], b[TN];
#pragma unroll
            for (int x = 0; x < TM; ++x) a[x] = *(const f4*)(Xs + abase[x] + toff);
#pragma unroll
            for (int y = 0; y < TN; ++y)
                b[y] = *(const f4*)(Ws + (((wn * TN + y) * 16 + li) * RS + tap) * LDW + gi * 4);
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int x = 0; x < TM; ++x)
#pragma unroll
                    for (int y = 0; y < TN; ++y) acc[x][y] = mfma16x16x4(a[x][j], b[y][j], acc[x][y]);
        }
    };
    if (ntot <= NU * 256) {
        const float* sp[NU];
        int d[NU];
        f4 v[NU];
#pragma unroll
        for (int u = 0; u < NU; ++u) {
            decode(tid + u * 256, sp[u], d[u]);
            v[u] = sp[u] ? *(const f4*)sp[u] : f4{0.f, 0.f, 0.f, 0.f};
        }
        for (int cgp = 0; cgp < ngroups; ++cgp) {
#pragma unroll
            for (int u = 0; u < NU; ++u)
                if (d[u] >= 0)
                    *(f4*)(lds + d[u]) = (INBN && sp[u] && tid + u * 256 < nx) ? fold(v[u], cgp * 16 + q * 4) : v[u];
            __syncthreads();
            if (cgp + 1 < ngroups) {
                const int c1 = (cgp + 1) * 16;
#pragma unroll
                for (int u = 0; u < NU; ++u) v[u] = sp[u] ? *(const f4*)(sp[u] + c1) : f4{0.f, 0.f, 0.f, 0.f};
            }
            compute();
            __syncthreads();
        }
    } else {
        for (int cgp = 0; cgp < ngroups; ++cgp) {
            const int c0 = cgp * 16;
            for (int base = tid; base < ntot; base += NU * 256) {
                // all of the batch's loads first (elements without a source
                // load the source's first quad, a valid address, and are
                // zeroed afterwards): with a conditional load and the fold
                // right behind each, they would go out one at a time
                f4 v[NU];
                int d[NU];
                bool z[NU];
#pragma unroll
                for (int u = 0; u < NU; ++u) {
                    const float* sp;
                    decode(base + u * 256, sp, d[u]);
                    z[u] = !sp;
                    v[u] = ld_global4((sp ? sp : src + q * 4) + c0);
                }
#pragma unroll
                for (int u = 0; u < NU; ++u) {
                    if (z[u]) v[u] = f4{0.f, 0.f, 0.f, 0.f};
                    else if (INBN && base + u * 256 < nx) v[u] = fold(v[u], c0 + q * 4);
                }
#pragma unroll
                for (int u = 0; u < NU; ++u)
                    if (d[u] >= 0) *(f4*)(lds + d[u]) = v[u];
            }
            __syncthreads();
            compute();
            __syncthreads();
        }
    }

    const long m0 = (long)blockIdx.x * TP;      // tiles are consecutive runs of the NHWC rows
    const int pix_base = wm * TM * 16;
    const int n_base = n0 + wn * TN * 16;
    f4 bs0 = f4{0.f, 0.f, 0.f, 0.f}, bs1 = bs0;   // data gradient with STATS: sum gm, sum gm*xhat
    if (bias) {
#pragma unroll
        for (int y = 0; y < TN; ++y) {
            const int n = n_base + y * 16 + li;
            const float bb = n < g.Ncols ? bias[n] : 0.f;
#pragma unroll
            for (int x = 0; x < TM; ++x)
#pragma unroll
                for (int i = 0; i < 4; ++i) acc[x][y][i] += bb;
        }
    }
    // the wave's TM*16 x TN*16 output block, transposed through LDS (the
    // X/W tiles are dead) so that every lane stores whole float4 channel
    // quads of one pixel
    {
        constexpr int OP = TN * 16 + 4;           // LDS pitch of a pixel row
        float* Ot = lds + wave * (TM * 16 * OP);
#pragma unroll
        for (int x = 0; x < TM; ++x)
#pragma unroll
            for (int y = 0; y < TN; ++y)
#pragma unroll
                for (int i = 0; i < 4; ++i) Ot[(x * 16 + gi * 4 + i) * OP + y * 16 + li] = acc[x][y][i];
        __builtin_amdgcn_wave_barrier();          // a wave's LDS accesses execute in order
        constexpr int QPP = TN * 4;               // float4 quads per pixel of the block
        // data gradient with STATS: this lane's channel quad is fixed (64 %
        // QPP == 0); its BN's mean, rstd, scale and shift
        f4 bmu{}, brs{}, bsc{}, bsh{};
        if (MODE == CONV_DGRAD && STATS) {
            const int n = n_base + (lane % QPP) * 4;
            if (n < g.Ncols) {
                bmu = *(const f4*)(bs.aux + n);
                brs = *(const f4*)(bs.aux + g.Ncols + n);
                bsc = *(const f4*)(bs.aux + 2 * g.Ncols + n);
                bsh = *(const f4*)(bs.aux + 3 * g.Ncols + n);
            }
        }
#pragma unroll
        for (int k = 0; k < TM * 16 * QPP / 64; ++k) {
            const int e = k * 64 + lane;
            const int p = e / QPP, qd = e - (e / QPP) * QPP;
            const int n = n_base + qd * 4;
            if (n < g.Ncols) {
                const f4 v = *(const f4*)(Ot + p * OP + qd * 4);
                f4* o = (f4*)(Y + (m0 + pix_base + p) * g.Ncols + n);
                const f4 tot = accumulate == kStoreAdd ? *o + v : (accumulate == kStoreRelu ? relu4(v) : v);
                *o = tot;
                if (MODE == CONV_DGRAD && STATS) {
                    // gm = the stored gradient where the forward's ReLU passed
                    // (its output y > 0, or fma(x, scale, shift) > 0), xhat of the BN input
                    const long e = (m0 + pix_base + p) * g.Ncols + n;
                    const f4 x = *(const f4*)(bs.x1 + e);
                    const f4 yv = bs.y ? *(const f4*)(bs.y + e) : f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const bool pass = bs.y ? yv[j] > 0.f : __builtin_fmaf(x[j], bsc[j], bsh[j]) > 0.f;
                        const float gm = pass ? tot[j] : 0.f;
                        bs0[j] += gm;
                        bs1[j] += gm * ((x[j] - bmu[j]) * brs[j]);
                    }
                }
            }
        }
    }
    if constexpr (MODE == CONV_DGRAD && STATS) {
        // lanes of one channel quad (lane mod QPP) summed by a fixed xor tree,
        // then the WM waves of this channel block in order
        constexpr int QPP = TN * 4;
        static_assert(64 % QPP == 0, "a lane keeps one channel quad");
#pragma unroll
        for (int o = QPP; o < 64; o <<= 1) {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                bs0[j] += __shfl_xor(bs0[j], o);
                bs1[j] += __shfl_xor(bs1[j], o);
            }
        }
        __shared__ f4 bred[4][2][QPP];
        if (lane < QPP) {
            bred[wave][0][lane] = bs0;
            bred[wave][1][lane] = bs1;
        }
        __syncthreads();
        if (threadIdx.x < WN * QPP) {
            const int wnb = threadIdx.x / QPP, qd = threadIdx.x - wnb * QPP;
            f4 t0 = bred[wnb * WM][0][qd], t1 = bred[wnb * WM][1][qd];
            for (int w = 1; w < WM; ++w) {
                t0 += bred[wnb * WM + w][0][qd];
                t1 += bred[wnb * WM + w][1][qd];
            }
            const int nb = n0 + wnb * TN * 16 + qd * 4;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int c = nb + j;
                if (c >= g.Ncols) continue;
                if (sums.acc) {
                    acc_add(sums.acc, 0, (int)blockIdx.x, g.Ncols, c, (double)t0[j]);
                    acc_add(sums.acc, 1, (int)blockIdx.x, g.Ncols, c, (double)t1[j]);
                } else {
                    sums.p0[(long)blockIdx.x * g.Ncols + c] = t0[j];
                    sums.p1[(long)blockIdx.x * g.Ncols + c] = t1[j];
                }
            }
        }
    }
    if constexpr (MODE == CONV_FWD && STATS) {
        // (every pixel of a tile lies inside the tensor)
        __shared__ float red[WM][3][BN];
        tile_moments<TM, TN, WM, BN, true>(
            acc, wm, wn, [](int, int) { return true; }, red,
            [&](int t, float n, float mu, float m2) {
                if (n0 + t < g.Ncols) tile_moments_store(sums, (int)blockIdx.x, g.Ncols, n0 + t, n, mu, m2);
            });
    }
}

// Picks (WM, TM, TN) and the tile rows OH for the spatial kernel, or returns
// false when no shape fits (the GEMM-style kernels take those passes).
struct TileCfg { int wm, tm, tn; TileGeom t; size_t lds; };
static bool pick_tile(int mode, const ConvGeom& g, TileCfg& out) {
    if (g.Cs % 16 != 0 || g.Ncols % 4 != 0) return false;
    if (!((g.R == 3 && g.S == 3) || (g.R == 1 && g.S == 1))) return false;
    if (mode == CONV_DGRAD && g.stride != 1) return false;
    static const int cands[][3] = {
        // wm, tm, tn  (tile pixels = wm*tm*16, output channels = (4/wm)*tn*16)
        {4, 4, 1}, {4, 2, 1}, {2, 4, 1}, {2, 2, 1}, {1, 4, 1}, {2, 2, 2}, {1, 4, 2}, {4, 1, 1}, {2, 1, 1}, {1, 2, 1},
        {1, 1, 1}};
    const long M = (long)g.Nb * g.Ho * g.Wo;
    // first choice: four waves along the pixels, 16 output channels, and a
    // tile of 8 output rows (4 for strided passes) -- measured fastest at
    // ResNet-20's shapes (32x32, 16x16 and 8x8 outputs)
    int pref[3] = {0, 0, 0};
    const int prow = g.stride == 1 ? 8 : 4;
    if ((prow * g.Wo) % 64 == 0) {
        const int tm = prow * g.Wo / 64;
        if (tm == 1 || tm == 2 || tm == 4) pref[0] = 4, pref[1] = tm, pref[2] = 1;
    }
    for (int ci = -1; ci < (int)(sizeof(cands) / sizeof(cands[0])); ++ci) {
        const int* c = ci < 0 ? pref : cands[ci];
        if (!c[0]) continue;
        const int wm = c[0], tm = c[1], tn = c[2];
        const int tp = wm * tm * 16, bn = (4 / wm) * tn * 16;
        if (bn > 16 && g.Ncols <= bn / 2) continue;             // output width too small for this tile
        if (g.Ncols > 16 && bn == 16 && g.Ncols % 32 == 0 && wm != 4) continue;
        if (tp % g.Wo) continue;
        const int oh = tp / g.Wo;
        if (oh < 1 || g.Ho % oh) continue;
        const int pad_eff = mode == CONV_FWD ? g.pad : g.R - 1 - g.pad;
        const int ih = (oh - 1) * g.stride + g.R, iw = (g.Wo - 1) * g.stride + g.S;
        // staged X and W tiles; the epilogue's transpose reuses the space
        const size_t lds = sizeof(float) * std::max<size_t>(20 * ((size_t)ih * iw + (size_t)bn * g.R * g.S),
                                                            (size_t)4 * tm * 16 * (tn * 16 + 4));
        if (lds > 60 * 1024) continue;   // leaves room for the static statistics arrays
        const long tiles = M / tp;
        if (tiles * ((g.Ncols + bn - 1) / bn) < 128) continue;
        const unsigned inv = (unsigned)((0x100000000ull + iw - 1) / iw);
        out = {wm, tm, tn, {oh, ih, iw, pad_eff, g.Ho / oh, inv}, lds};
        return true;
    }
    return false;
}

template <int MODE, int KS, int WM, int TM, int TN>
static hipError_t launch_tile(const float* src, const float* B, const float* bias, float* Y, const ConvGeom& g,
                              const TileCfg& c, int acc, const BnSums* stats, const BnFwd* inbn,
                              const BnBwdSum* bsv, hipStream_t st) {
    constexpr int BN = (4 / WM) * TN * 16;
    dim3 grid((unsigned)(g.Nb * c.t.tiles_per_img), (unsigned)((g.Ncols + BN - 1) / BN));
    const BnSums sm = stats ? *stats : BnSums{};
    const BnFwd ib = inbn ? *inbn : BnFwd{};
    const BnBwdSum bsum = bsv ? *bsv : BnBwdSum{};
    // a data gradient's statistics are the sums of a BN backward (bsv)
    if (MODE == CONV_DGRAD && stats && (!bsv || (acc && !bsv->y))) return hipErrorInvalidValue;
    if (inbn) {
        if (MODE != CONV_FWD || g.Cs > kFoldMaxC) return hipErrorInvalidValue;
        if (stats)
            launch((conv_tile_f32<MODE, KS, WM, TM, TN, true, true>), grid, dim3(256), c.lds, st, src, B, bias, Y, g,
                   c.t, (int)acc, sm, ib, bsum);
        else
            launch((conv_tile_f32<MODE, KS, WM, TM, TN, false, true>), grid, dim3(256), c.lds, st, src, B, bias, Y, g,
                   c.t, (int)acc, sm, ib, bsum);
    } else if (stats) {
        launch((conv_tile_f32<MODE, KS, WM, TM, TN, true, false>), grid, dim3(256), c.lds, st, src, B, bias, Y, g,
               c.t, (int)acc, sm, ib, bsum);
    } else {
        launch((conv_tile_f32<MODE, KS, WM, TM, TN, false, false>), grid, dim3(256), c.lds, st, src, B, bias, Y, g,
               c.t, (int)acc, sm, ib, bsum);
    }
    return hipGetLastError();
}

template <int MODE>
static hipError_t dispatch_tile(const float* src, const float* B, const float* bias, float* Y, const ConvGeom& g,
                                const TileCfg& c, int acc, const BnSums* stats, const BnFwd* inbn,
                                const BnBwdSum* bsv, hipStream_t st) {
#define TILE(WM_, TM_, TN_)                                                                                        \
    if (c.wm == WM_ && c.tm == TM_ && c.tn == TN_) {                                                               \
        if (g.R == 3) return launch_tile<MODE, 3, WM_, TM_, TN_>(src, B, bias, Y, g, c, acc, stats, inbn, bsv, st); \
        return launch_tile<MODE, 1, WM_, TM_, TN_>(src, B, bias, Y, g, c, acc, stats, inbn, bsv, st);               \
    }
    TILE(4, 4, 1) TILE(4, 2, 1) TILE(2, 4, 1) TILE(2, 2, 1) TILE(1, 4, 1) TILE(2, 2, 2) TILE(1, 4, 2)
    TILE(4, 1, 1) TILE(2, 1, 1) TILE(1, 2, 1) TILE(1, 1, 1)
#undef TILE
    return hipErrorInvalidValue;
}

// Data gradient of a stride-2 conv, split by output parity.  dX pixel
// (2i + a, 2j + b) only receives taps (r, s) with a + pad - r and b + pad - s
// even, from dY[i + (a + pad - r)/2][j + (b + pad - s)/2]: per parity class
// (a, b) this is a dense stride-1 correlation over dY with a subset of the
// taps (3x3, pad 1: 1, 2, 2 and 4 taps; 1x1, pad 0: one tap, class (0, 0)).
// A workgroup takes OH class rows of one image for all four classes (a dX
// tile of 2 OH rows), so every workgroup runs all R*S taps once and the dY
// rows it reads are staged in LDS once per 16 dY channels; no MFMA is spent
// on taps that fall between strides.  The finished tile is transposed
// through LDS and stored as float4 channel quads.
struct S2Geom { int OH, IH, IW, Hc, Wc, tiles_per_img, dr0, ds0; unsigned IW_inv; };

template <int KS, int PAD, int WM, int TM, int TN>
__global__ __launch_bounds__(256) void conv_dgrad_s2_f32(const float* __restrict__ dY, const float* __restrict__ B,
                                                         float* __restrict__ dX, ConvGeom g, S2Geom t,
                                                         int accumulate) {
    constexpr int WN = 4 / WM;
    constexpr int TP = WM * TM * 16, BN = WN * TN * 16;
    constexpr int LDW = 20;
    constexpr int RS = KS * KS;
    constexpr int NU = 8;
    extern __shared__ float lds[];
    float* Xs = lds;                              // [IH*IW][LDW] dY rows
    float* Ws = lds + t.IH * t.IW * LDW;          // [BN][RS][LDW]
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave % WM, wn = wave / WM;
    const int gi = lane >> 4, li = lane & 15;
    const int img = blockIdx.x / t.tiles_per_img;
    const int i0 = (blockIdx.x - img * t.tiles_per_img) * t.OH;
    const int n0 = blockIdx.y * BN;
    const int h_org = i0 + t.dr0, w_org = t.ds0;

    int abase[TM];
#pragma unroll
    for (int x = 0; x < TM; ++x) {
        const int p = (wm * TM + x) * 16 + li;
        const int oh = p / t.Wc, ow = p - (p / t.Wc) * t.Wc;
        abase[x] = (oh * t.IW + ow) * LDW + gi * 4;
    }
    f4 acc[4][TM][TN];
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) acc[c][i][j] = f4{0.f, 0.f, 0.f, 0.f};

    const int q = tid & 3;
    const int nx = t.IH * t.IW * 4, ntot = nx + BN * RS * 4;
    auto decode = [&](int e, const float*& sp, int& d) {
        sp = nullptr;
        d = -1;
        if (e < nx) {
            const int pix = e >> 2;
            const int ih = (int)__umulhi((unsigned)pix, t.IW_inv);
            const int iw = pix - ih * t.IW;
            const int h = h_org + ih, w = w_org + iw;
            if (h >= 0 && h < g.Hs && w >= 0 && w < g.Ws)
                sp = dY + ((long)(img * g.Hs + h) * g.Ws + w) * g.Cs + q * 4;
            d = pix * LDW + q * 4;
        } else if (e < ntot) {
            const int rest = (e - nx) >> 2;
            const int tap = rest % RS, nl = rest / RS;
            const int n = n0 + nl;
            if (n < g.Ncols) sp = B + ((long)n * RS + tap) * g.Cs + q * 4;
            d = t.IH * t.IW * LDW + rest * LDW + q * 4;
        }
    };
    auto compute = [&]() {
#pragma unroll
        for (int cls = 0; cls < 4; ++cls) {
            const int ca = cls >> 1, cb = cls & 1;
#pragma unroll
            for (int r = 0; r < KS; ++r)
#pragma unroll
                for (int sx = 0; sx < KS; ++sx) {
                    if (((ca + PAD - r) & 1) || ((cb + PAD - sx) & 1)) continue;
                    // source row i + (a + pad - r)/2, column j + (b + pad - s)/2
                    const int dr = (ca + PAD - r) / 2 - t.dr0, ds = (cb + PAD - sx) / 2 - t.ds0;
                    const int toff = (dr * t.IW + ds) * LDW;
                    const int tap = r * KS + sx;
                    f4 av[TM], bv[TN];
#pragma unroll
                    for (int x = 0; x < TM; ++x) av[x] = *(const f4*)(Xs + abase[x] + toff);
#pragma unroll
                    for (int y = 0; y < TN; ++y)
                        bv[y] = *(const f4*)(Ws + (((wn * TN + y) * 16 + li) * RS + tap) * LDW + gi * 4);
#pragma unroll
                    for (int j = 0; j < 4; ++j)
#pragma unroll
                        for (int x = 0; x < TM; ++x)
#pragma unroll
                            for (int y = 0; y < TN; ++y)
                                acc[cls][x][y] = mfma16x16x4(av[x][j], bv[y][j], acc[cls][x][y]);
                }
        }
    };
    const int ngroups = g.Cs >> 4;
    if (ntot <= NU * 256) {
        const float* sp[NU];
        int d[NU];
        f4 v[NU];
#pragma unroll
        for (int u = 0; u < NU; ++u) {
            decode(tid + u * 256, sp[u], d[u]);
            v[u] = sp[u] ? *(const f4*)sp[u] : f4{0.f, 0.f, 0.f, 0.f};
        }
        for (int cgp = 0; cgp < ngroups; ++cgp) {
#pragma unroll
            for (int u = 0; u < NU; ++u)
                if (d[u] >= 0) *(f4*)(lds + d[u]) = v[u];
            __syncthreads();
            if (cgp + 1 < ngroups) {
                const int c1 = (cgp + 1) * 16;
#pragma unroll
                for (int u = 0; u < NU; ++u) v[u] = sp[u] ? *(const f4*)(sp[u] + c1) : f4{0.f, 0.f, 0.f, 0.f};
            }
            compute();
            __syncthreads();
        }
    } else {
        for (int cgp = 0; cgp < ngroups; ++cgp) {
            const int c0 = cgp * 16;
            for (int base = tid; base < ntot; base += NU * 256) {
                f4 v[NU];
                int d[NU];
#pragma unroll
                for (int u = 0; u < NU; ++u) {
                    const float* sp;
                    decode(base + u * 256, sp, d[u]);
                    v[u] = sp ? *(const f4*)(sp + c0) : f4{0.f, 0.f, 0.f, 0.f};
                }
#pragma unroll
                for (int u = 0; u < NU; ++u)
                    if (d[u] >= 0) *(f4*)(lds + d[u]) = v[u];
            }
            __syncthreads();
            compute();
            __syncthreads();
        }
    }

    // the dX tile (2 OH rows x 2 Wc columns x BN channels) in LDS, pixel-major
    constexpr int OP = BN + 4;
    const int tw = 2 * t.Wc;
#pragma unroll
    for (int cls = 0; cls < 4; ++cls)
#pragma unroll
        for (int x = 0; x < TM; ++x)
#pragma unroll
            for (int y = 0; y < TN; ++y)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int p = (wm * TM + x) * 16 + gi * 4 + i;
                    const int oh = p / t.Wc, ow = p - (p / t.Wc) * t.Wc;
                    const int tp = (2 * oh + (cls >> 1)) * tw + 2 * ow + (cls & 1);
                    lds[tp * OP + (wn * TN + y) * 16 + li] = acc[cls][x][y][i];
                }
    __syncthreads();
    constexpr int QPP = BN / 4;
    for (int e = tid; e < 4 * TP * QPP; e += 256) {
        const int tp = e / QPP, qd = e - (e / QPP) * QPP;
        const int n = n0 + qd * 4;
        if (n >= g.Ncols) continue;
        const int hr = tp / tw, wc = tp - (tp / tw) * tw;
        const f4 v = *(const f4*)(lds + tp * OP + qd * 4);
        f4* o = (f4*)(dX + ((long)(img * g.Ho + 2 * i0 + hr) * g.Wo + wc) * g.Ncols + n);
        *o = accumulate == kStoreAdd ? *o + v : (accumulate == kStoreRelu ? relu4(v) : v);
    }
}

// Tile shape of the parity-split stride-2 data gradient, or false when it
// does not apply.
struct S2Cfg { int wm, tm, tn; S2Geom t; size_t lds; };
static bool pick_s2(const ConvGeom& g, S2Cfg& out) {
    if (g.stride != 2 || g.Cs % 16 || g.Ncols % 4 || (g.Ho & 1) || (g.Wo & 1)) return false;
    if (!((g.R == 3 && g.S == 3 && g.pad == 1) || (g.R == 1 && g.S == 1 && g.pad == 0))) return false;
    const int Hc = g.Ho / 2, Wc = g.Wo / 2;
    // source offsets (a + pad - r)/2 over every class and tap
    int dr0 = 1 << 20, dr1 = -(1 << 20);
    for (int a = 0; a < 2; ++a)
        for (int r = 0; r < g.R; ++r)
            if (((a + g.pad - r) & 1) == 0) {
                dr0 = std::min(dr0, (a + g.pad - r) / 2);
                dr1 = std::max(dr1, (a + g.pad - r) / 2);
            }
    static const int cands[][3] = {{4, 4, 1}, {4, 2, 1}, {4, 1, 1}, {2, 2, 1}, {2, 1, 1}, {1, 1, 1}};
    for (int pass = 0; pass < 2; ++pass)
        for (auto& c : cands) {
            const int wm = c[0], tm = c[1], tn = c[2];
            const int tp = wm * tm * 16, bn = (4 / wm) * tn * 16;
            if (bn > 16 && g.Ncols <= bn / 2) continue;
            if (tp % Wc) continue;
            const int oh = tp / Wc;
            if (oh < 1 || Hc % oh) continue;
            const long wgs = (long)g.Nb * (Hc / oh) * ((g.Ncols + bn - 1) / bn);
            if (pass == 0 && wgs < 256) continue;     // first look for shapes that fill the chip
            const int ih = oh + dr1 - dr0, iw = Wc + dr1 - dr0;
            const size_t lds = sizeof(float) * std::max<size_t>(20 * ((size_t)ih * iw + (size_t)bn * g.R * g.S),
                                                                (size_t)4 * tp * (bn + 4));
            if (lds > 60 * 1024) continue;
            const unsigned inv = (unsigned)((0x100000000ull + iw - 1) / iw);
            out = {wm, tm, tn, {oh, ih, iw, Hc, Wc, Hc / oh, dr0, dr0, inv}, lds};
            return true;
        }
    return false;
}

template <int KS, int PAD, int WM, int TM, int TN>
static hipError_t launch_s2(const float* dY, const float* B, float* dX, const ConvGeom& g, const S2Cfg& c, int acc,
                            hipStream_t st) {
    constexpr int BN = (4 / WM) * TN * 16;
    dim3 grid((unsigned)(g.Nb * c.t.tiles_per_img), (unsigned)((g.Ncols + BN - 1) / BN));
    launch((conv_dgrad_s2_f32<KS, PAD, WM, TM, TN>), grid, dim3(256), c.lds, st, dY, B, dX, g, c.t,
                       (int)acc);
    return hipGetLastError();
}

static hipError_t dispatch_s2(const float* dY, const float* B, float* dX, const ConvGeom& g, const S2Cfg& c, int acc,
                              hipStream_t st) {
#define S2(WM_, TM_, TN_)                                                                              \
    if (c.wm == WM_ && c.tm == TM_ && c.tn == TN_) {                                                   \
        if (g.R == 3) return launch_s2<3, 1, WM_, TM_, TN_>(dY, B, dX, g, c, acc, st);                 \
        return launch_s2<1, 0, WM_, TM_, TN_>(dY, B, dX, g, c, acc, st);                               \
    }
    S2(4, 4, 1) S2(4, 2, 1) S2(4, 1, 1) S2(2, 2, 1) S2(2, 1, 1) S2(1, 1, 1)
#undef S2
    return hipErrorInvalidValue;
}

template <int MODE, int WM, int TM, int TN>
static hipError_t launch_cfg(const float* src, const float* B, const float* bias, float* Y, const ConvGeom& g,
                             int acc, const BnSums* stats, hipStream_t st) {
    constexpr int BM = WM * TM * 16, BN = (4 / WM) * TN * 16;
    const long M = (long)g.Nb * g.Ho * g.Wo;
    dim3 grid((unsigned)((M + BM - 1) / BM), (unsigned)((g.Ncols + BN - 1) / BN));
    const bool fast = g.Cs % 16 == 0;
    if (stats) {
        if (fast)
            launch((conv_igemm_f32<MODE, WM, TM, TN, true, true>), grid, dim3(256), 0, st, src, B, bias,
                               Y, g, (int)acc, stats ? *stats : BnSums{});
        else
            launch((conv_igemm_f32<MODE, WM, TM, TN, false, true>), grid, dim3(256), 0, st, src, B, bias,
                               Y, g, (int)acc, stats ? *stats : BnSums{});
    } else {
        if (fast)
            launch((conv_igemm_f32<MODE, WM, TM, TN, true, false>), grid, dim3(256), 0, st, src, B, bias,
                               Y, g, (int)acc, stats ? *stats : BnSums{});
        else
            launch((conv_igemm_f32<MODE, WM, TM, TN, false, false>), grid, dim3(256), 0, st, src, B, bias,
                               Y, g, (int)acc, stats ? *stats : BnSums{});
    }
    return hipGetLastError();
}

// Tile configuration.  Cs % 16 == 0 uses the LDS kernel with (BM, BN, WM)
// by output width and rows; other passes (the padded image) the direct one.
struct ConvCfg { int lds, bm, bn, wm, tm, tn; };
static ConvCfg pick_cfg(const ConvGeom& g) {
    const long M = (long)g.Nb * g.Ho * g.Wo;
    if (g.Cs % 16 == 0) {
        if (g.Ncols <= 16) return {1, M >= 256L * 256 ? 256 : 64, 16, 4, 0, 0};
        if (g.Ncols <= 32) return {1, M >= 128L * 256 ? 128 : 64, 32, M >= 128L * 256 ? 4 : 2, 0, 0};
        if (g.Ncols <= 64) return {1, M >= 64L * 256 ? 64 : 32, 64, M >= 64L * 256 ? 2 : 1, 0, 0};
        return {1, 64, 128, 2, 0, 0};
    }
    if (g.Ncols <= 16) return {0, 128, 16, 4, 2, 1};
    if (g.Ncols <= 32) return {0, 128, 32, 4, 2, 2};
    if (g.Ncols <= 64 || M < 64L * 512) {
        if (M >= 64L * 512) return {0, 64, 64, 2, 2, 2};
        return {0, 32, 64, 2, 1, 2};
    }
    return {0, 64, 128, 2, 2, 4};
}

template <int MODE>
static hipError_t launch_mode(const float* src, const float* B, const float* bias, float* Y, const ConvGeom& g,
                              int acc, const BnSums* stats, const BnFwd* inbn, const BnBwdSum* bsv, hipStream_t st) {
    TileCfg tc;
    if (pick_tile(MODE, g, tc)) return dispatch_tile<MODE>(src, B, bias, Y, g, tc, acc, stats, inbn, bsv, st);
    if (inbn || bsv) return hipErrorInvalidValue;   // folding and backward sums need the spatial kernel
    if (MODE == CONV_DGRAD) {
        S2Cfg sc;
        if (pick_s2(g, sc)) return dispatch_s2(src, B, Y, g, sc, acc, st);
    }
    ConvCfg c = pick_cfg(g);
    if (c.lds) {
        if (c.bn == 16) {
            if (c.bm == 256) return launch_lds<MODE, 256, 16, 4>(src, B, bias, Y, g, acc, stats, st);
            return launch_lds<MODE, 64, 16, 4>(src, B, bias, Y, g, acc, stats, st);
        }
        if (c.bn == 32) {
            if (c.bm == 128) return launch_lds<MODE, 128, 32, 4>(src, B, bias, Y, g, acc, stats, st);
            return launch_lds<MODE, 64, 32, 2>(src, B, bias, Y, g, acc, stats, st);
        }
        if (c.bn == 64) {
            if (c.bm == 64) return launch_lds<MODE, 64, 64, 2>(src, B, bias, Y, g, acc, stats, st);
            return launch_lds<MODE, 32, 64, 1>(src, B, bias, Y, g, acc, stats, st);
        }
        return launch_lds<MODE, 64, 128, 2>(src, B, bias, Y, g, acc, stats, st);
    }
    if (c.wm == 4 && c.tn == 1) return launch_cfg<MODE, 4, 2, 1>(src, B, bias, Y, g, acc, stats, st);
    if (c.wm == 4) return launch_cfg<MODE, 4, 2, 2>(src, B, bias, Y, g, acc, stats, st);
    if (c.tn == 4) return launch_cfg<MODE, 2, 2, 4>(src, B, bias, Y, g, acc, stats, st);
    if (c.tm == 2) return launch_cfg<MODE, 2, 2, 2>(src, B, bias, Y, g, acc, stats, st);
    return launch_cfg<MODE, 2, 1, 2>(src, B, bias, Y, g, acc, stats, st);
}

int conv_tile_rows(const ConvGeom& g) {
    TileCfg t;
    if (pick_tile(CONV_FWD, g, t)) return t.wm * t.tm * 16;
    return pick_cfg(g).bm;
}

hipError_t launch_conv_igemm(int mode, const float* src, const float* B, const float* bias, float* Y,
                             const ConvGeom& g, int accumulate, const BnSums* stats, hipStream_t st,
                             const BnFwd* inbn, const BnBwdSum* bsum) {
    if (mode == CONV_FWD) {
        if (bsum) return hipErrorInvalidValue;
        return launch_mode<CONV_FWD>(src, B, bias, Y, g, accumulate, stats, inbn, nullptr, st);
    }
    if (inbn || (bsum != nullptr) != (stats != nullptr)) return hipErrorInvalidValue;
    return launch_mode<CONV_DGRAD>(src, B, bias, Y, g, accumulate, stats, nullptr, bsum, st);
}

int conv_dgrad_sum_tiles(const ConvGeom& gd) {
    TileCfg tc;
    if (!pick_tile(CONV_DGRAD, gd, tc)) return 0;
    return gd.Nb * tc.t.tiles_per_img;
}

bool conv_fold_ok(const ConvGeom& g, const WgradPlan& p) {
    TileCfg tc;
    return g.Cs <= kFoldMaxC && p.tile && pick_tile(CONV_FWD, g, tc);
}

// ------------------------------------------------------------------------
// weight gradient
// ------------------------------------------------------------------------

struct WgArgs {
    int Nb, Hi, Wi, Cin_p, Ho, Wo, Cout, R, S, stride, pad, pix_per_split;
};

template <int TM, int TN>
__global__ __launch_bounds__(256) void conv_wgrad_f32(const float* __restrict__ dY, const float* __restrict__ X,
                                                      float* __restrict__ part, WgArgs a) {
    constexpr int BMw = TM * 16, BNw = TN * 16;
    constexpr int NA = 64 * (BMw / 4) / 256;   // dY quads per thread per chunk
    constexpr int NB = 64 * (BNw / 4) / 256;   // im2col quads per thread per chunk
    __shared__ float As[64][BMw + 4];
    __shared__ float Bs[64][BNw + 4];
    __shared__ float red[TM * TN * 4][64];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int gi = lane >> 4, li = lane & 15;
    const int HoWo = a.Ho * a.Wo;
    const int M = a.Nb * HoWo;
    const int Ktot = a.R * a.S * a.Cin_p;
    const int Cq = a.Cin_p >> 2;
    const int m0 = blockIdx.x * BMw, n0 = blockIdx.y * BNw;
    const int p_begin = blockIdx.z * a.pix_per_split;
    const int p_end = min(M, p_begin + a.pix_per_split);

    // each thread's column quad is the same in every chunk: decode it once
    const int bcq = tid % (BNw / 4);
    const int col = n0 + bcq * 4;
    const bool col_ok = col < Ktot;
    int br = 0, bs = 0, bc = 0;
    if (col_ok) {
        const int quad = col >> 2;
        const int tap = quad / Cq;
        bc = (quad - tap * Cq) * 4;
        br = tap / a.S;
        bs = tap - br * a.S;
    }
    const int acq = tid % (BMw / 4);
    const int aco = m0 + acq * 4;

    f4 ra[NA], rb[NB];
    auto load = [&](int pc) {
#pragma unroll
        for (int k = 0; k < NA; ++k) {
            const int px = (tid + 256 * k) / (BMw / 4);
            const int p = pc + px;
            ra[k] = (p < p_end && aco < a.Cout) ? *(const f4*)(dY + (long)p * a.Cout + aco) : f4{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
        for (int k = 0; k < NB; ++k) {
            const int px = (tid + 256 * k) / (BNw / 4);
            const int p = pc + px;
            f4 v = f4{0.f, 0.f, 0.f, 0.f};
            if (p < p_end && col_ok) {
                const int n = p / HoWo;
                const int rem = p - n * HoWo;
                const int ho = rem / a.Wo, wo = rem - ho * a.Wo;
                const int hi = ho * a.stride - a.pad + br, wi = wo * a.stride - a.pad + bs;
                if (hi >= 0 && hi < a.Hi && wi >= 0 && wi < a.Wi)
                    v = *(const f4*)(X + ((long)(n * a.Hi + hi) * a.Wi + wi) * a.Cin_p + bc);
            }
            rb[k] = v;
        }
    };

    f4 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};

    if (p_begin < p_end) load(p_begin);
    for (int pc = p_begin; pc < p_end; pc += 64) {
#pragma unroll
        for (int k = 0; k < NA; ++k) *(f4*)&As[(tid + 256 * k) / (BMw / 4)][acq * 4] = ra[k];
#pragma unroll
        for (int k = 0; k < NB; ++k) *(f4*)&Bs[(tid + 256 * k) / (BNw / 4)][bcq * 4] = rb[k];
        __syncthreads();
        if (pc + 64 < p_end) load(pc + 64);   // next chunk in flight during this one's MFMAs
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int row = 16 * wave + 4 * j + gi;
            float av[TM], bv[TN];
#pragma unroll
            for (int t = 0; t < TM; ++t) av[t] = As[row][t * 16 + li];
#pragma unroll
            for (int t = 0; t < TN; ++t) bv[t] = Bs[row][t * 16 + li];
#pragma unroll
            for (int x = 0; x < TM; ++x)
#pragma unroll
                for (int y = 0; y < TN; ++y) acc[x][y] = mfma16x16x4(av[x], bv[y], acc[x][y]);
        }
        __syncthreads();
    }

    // waves 0..3 summed in order through LDS
    for (int w = 0; w < 4; ++w) {
        if (wave == w) {
#pragma unroll
            for (int x = 0; x < TM; ++x)
#pragma unroll
                for (int y = 0; y < TN; ++y)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        float* slot = &red[(x * TN + y) * 4 + i][lane];
                        *slot = (w == 0) ? acc[x][y][i] : *slot + acc[x][y][i];
                    }
        }
        __syncthreads();
    }
    if (wave == 3) {
        float* out = part + (long)blockIdx.z * a.Cout * Ktot;
#pragma unroll
        for (int x = 0; x < TM; ++x)
#pragma unroll
            for (int y = 0; y < TN; ++y) {
                const int cc = n0 + y * 16 + li;
                if (cc >= Ktot) continue;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int co = m0 + x * 16 + gi * 4 + i;
                    if (co < a.Cout) out[(long)co * Ktot + cc] = red[(x * TN + y) * 4 + i][lane];
                }
            }
    }
}

// Spatially tiled weight gradient (Cs % 16 == 0): a workgroup takes a tile
// of TP output pixels (OH full rows of one image, or IMGS whole images), 16
// output channels and 16 input channels, and produces the partial
//     dW[co][r][s][c] = sum over the tile's pixels p of dY[p][co] * X[src(p, r, s)][c]
// for every tap.  The tile's input rows (halo and padding included; for a
// 1x1 conv just the pixels it reads) are staged in LDS once; each wave takes
// NG groups of 16 pixels, keeps their dY values in registers and runs all
// taps over them, so dY is read once and X once per channel block.  The
// reduction dimension k of v_mfma_f32_16x16x4_f32 is the pixel: lane
// (li, gi) supplies dY[p][co0 + li] and X[src(p)][c0 + li] for the same four
// pixels p = 16 g + 4 gi + j.  Waves are summed in a fixed order and every
// tile writes its own partial part[tile][co][(r, s, c)], summed in order by
// the reduce kernel.
struct WgTileGeom { int OH, IMGS, IH, IW, tiles_per_img, TP; unsigned IW_inv, IHW_inv; };

// Held to 128 registers (four waves per SIMD) where that needs no spilling:
// every variant but the strided 1x1 one.
template <int RS, int NG, int ST, bool K1>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu((RS == 9 || ST == 1) ? 4 : 1, 8)))
void conv_wgrad_tile_f32(const float* __restrict__ dY, const float* __restrict__ X,
                                                           float* __restrict__ part, WgArgs a, WgTileGeom t,
                                                           const float* __restrict__ in_ss) {
    constexpr int LDW = 20;
    constexpr int JST = (K1 ? 1 : ST) * LDW;   // LDS distance between a lane's four pixels
    constexpr int TP = NG * 64;
    constexpr int NU = 8;
    extern __shared__ float lds[];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int gi = lane >> 4, li = lane & 15;
    const int tile = blockIdx.x;
    const int co0 = blockIdx.y * 16, c0 = blockIdx.z * 16;
    const int img0 = t.IMGS == 1 ? tile / t.tiles_per_img : tile * t.IMGS;
    const int oh0 = t.IMGS == 1 ? (tile - img0 * t.tiles_per_img) * t.OH : 0;
    const int Ktot = RS * a.Cin_p;
    const long m0 = (long)tile * TP;
    const int ohw = t.OH * a.Wo;
    const int npix = t.IMGS * t.IH * t.IW;
    float* Xs = lds;                         // [npix][LDW] input rows of the tile
    float* Ds = lds + npix * LDW;            // [TP][LDW] dY of the tile, 16 channels

    // stage X rows and the dY tile: element e = tid + 256 u has quad tid & 3.
    // All of a batch's loads are issued before any value is used: elements
    // without a source (zero padding, past the tiles) load X's first quad of
    // the channel block, a valid address, and are zeroed afterwards (with
    // conditional loads and the fold right behind each, the loads would go
    // out one round trip at a time).
    {
        const int q = tid & 3;
        const int nx = npix * 4, ntot = nx + TP * 4;
        // the fold's scale and shift of this thread's channel quad (the same
        // for all its elements)
        float fsc[4] = {1.f, 1.f, 1.f, 1.f}, fsh[4] = {0.f, 0.f, 0.f, 0.f};
        if (in_ss) {
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                fsc[k] = in_ss[c0 + q * 4 + k];
                fsh[k] = in_ss[a.Cin_p + c0 + q * 4 + k];
            }
        }
        for (int base = tid; base < ntot; base += NU * 256) {
            f4 v[NU];
            int d[NU];
            bool z[NU];
#pragma unroll
            for (int u = 0; u < NU; ++u) {
                const int e = base + u * 256;
                const float* sp = X + c0 + q * 4;
                z[u] = true;
                d[u] = -1;
                if (e < nx) {
                    const int pix = e >> 2;
                    const int il = (int)__umulhi((unsigned)pix, t.IHW_inv);
                    const int rem = pix - il * (t.IH * t.IW);
                    const int ih = (int)__umulhi((unsigned)rem, t.IW_inv);
                    const int iw = rem - ih * t.IW;
                    const int h = K1 ? (oh0 + ih) * ST : oh0 * ST - a.pad + ih;
                    const int w = K1 ? iw * ST : iw - a.pad;
                    if (h >= 0 && h < a.Hi && w >= 0 && w < a.Wi) {
                        sp = X + ((long)((img0 + il) * a.Hi + h) * a.Wi + w) * a.Cin_p + c0 + q * 4;
                        z[u] = false;
                    }
                    d[u] = pix * LDW + q * 4;
                } else if (e < ntot) {
                    const int p = (e - nx) >> 2;
                    sp = dY + (m0 + p) * a.Cout + co0 + q * 4;
                    z[u] = false;
                    d[u] = (npix + p) * LDW + q * 4;
                }
                v[u] = ld_global4(sp);
            }
#pragma unroll
            for (int u = 0; u < NU; ++u) {
                if (z[u]) v[u] = f4{0.f, 0.f, 0.f, 0.f};
                // X read through a folded BN + ReLU (padding stays zero)
                else if (in_ss && base + u * 256 < nx) {
#pragma unroll
                    for (int k = 0; k < 4; ++k) v[u][k] = fmaxf(__builtin_fmaf(v[u][k], fsc[k], fsh[k]), 0.f);
                }
            }
#pragma unroll
            for (int u = 0; u < NU; ++u)
                if (d[u] >= 0) *(f4*)(lds + d[u]) = v[u];
        }
    }

    // this lane's pixels p = 16 (wave NG + g) + 4 gi + j: four consecutive
    // pixels of one output row (Wo % 4 == 0), so one LDS base per group
    int boff[NG];
#pragma unroll
    for (int g = 0; g < NG; ++g) {
        const int p = (wave * NG + g) * 16 + gi * 4;
        const int il = p / ohw, rem = p - il * ohw;
        const int ohl = rem / a.Wo, ow = rem - ohl * a.Wo;
        boff[g] = (K1 ? p : (il * t.IH + ohl * ST) * t.IW + ow * ST) * LDW + li;
    }
    int toff[RS];
#pragma unroll
    for (int k = 0; k < RS; ++k) toff[k] = K1 ? 0 : ((k / 3) * t.IW + k % 3) * LDW;
    __syncthreads();

    f4 acc[RS];
#pragma unroll
    for (int k = 0; k < RS; ++k) acc[k] = f4{0.f, 0.f, 0.f, 0.f};
    // per group: the four dY values and all RS x 4 X operands are read before
    // its MFMAs, the next group's reads are issued before this group's MFMAs
    float bv[2][RS][4];
    f4 av[2];
#pragma unroll
    for (int j = 0; j < 4; ++j) av[0][j] = Ds[(wave * NG * 16 + gi * 4 + j) * LDW + li];
#pragma unroll
    for (int k = 0; k < RS; ++k)
#pragma unroll
        for (int j = 0; j < 4; ++j) bv[0][k][j] = Xs[boff[0] + toff[k] + j * JST];
#pragma unroll
    for (int g = 0; g < NG; ++g) {
        if (g + 1 < NG) {
#pragma unroll
            for (int j = 0; j < 4; ++j) av[(g + 1) & 1][j] = Ds[(((wave * NG + g + 1) * 16) + gi * 4 + j) * LDW + li];
#pragma unroll
            for (int k = 0; k < RS; ++k)
#pragma unroll
                for (int j = 0; j < 4; ++j) bv[(g + 1) & 1][k][j] = Xs[boff[g + 1] + toff[k] + j * JST];
        }
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int k = 0; k < RS; ++k) acc[k] = mfma16x16x4(av[g & 1][j], bv[g & 1][k][j], acc[k]);
    }
    __syncthreads();   // the staged tiles are dead: their space takes the wave sums

    // each wave's RS x 16 x 16 block into its own LDS slice, then the four
    // slices summed in order
    float* red = lds;   // [4][RS][16 co][16 c]
#pragma unroll
    for (int k = 0; k < RS; ++k)
#pragma unroll
        for (int i = 0; i < 4; ++i) red[((wave * RS + k) * 16 + gi * 4 + i) * 16 + li] = acc[k][i];
    __syncthreads();
    float* out = part + (long)tile * a.Cout * Ktot;
    for (int e = tid; e < RS * 256; e += 256) {
        const int k = e >> 8, col = (e >> 4) & 15, c = e & 15;
        const float v = ((red[e] + red[RS * 256 + e]) + red[2 * RS * 256 + e]) + red[3 * RS * 256 + e];
        out[(long)(co0 + col) * Ktot + k * a.Cin_p + c0 + c] = v;
    }
}

// Tile shape for the spatially tiled weight gradient, or false when it does
// not apply (the GEMM-style kernel takes those passes).
static bool pick_wgrad_tile(int Nb, int Hi, int Wi, int Cin_p, int Ho, int Wo, int Cout, int R, int S, int stride,
                            int pad, WgTileGeom& t) {
    if (Cin_p % 16 || Cout % 16 || Wo % 4 || (stride != 1 && stride != 2)) return false;
    if (!((R == 3 && S == 3) || (R == 1 && S == 1 && pad == 0))) return false;
    const bool k1 = R == 1;
    for (int tp : {256, 128, 64}) {
        int oh, imgs;
        if (Ho * Wo >= tp) {
            if (tp % Wo) continue;
            oh = tp / Wo;
            if (Ho % oh) continue;
            imgs = 1;
        } else {
            if (tp % (Ho * Wo)) continue;
            oh = Ho;
            imgs = tp / (Ho * Wo);
            if (Nb % imgs) continue;
        }
        const int ih = k1 ? oh : (oh - 1) * stride + R, iw = k1 ? Wo : (Wo - 1) * stride + S;
        const size_t lds = sizeof(float) * std::max<size_t>(((size_t)imgs * ih * iw + tp) * 20, (size_t)4 * R * S * 256);
        if (lds > 60 * 1024) continue;
        const unsigned iw_inv = (unsigned)((0x100000000ull + iw - 1) / iw);
        const unsigned ihw_inv = (unsigned)((0x100000000ull + ih * iw - 1) / (ih * iw));
        t = WgTileGeom{oh, imgs, ih, iw, imgs == 1 ? Ho / oh : 0, tp, iw_inv, ihw_inv};
        return true;
    }
    return false;
}

WgradPlan wgrad_plan(int Nb, int Hi, int Wi, int Cin_p, int Ho, int Wo, int Cout, int R, int S, int stride, int pad) {
    WgradPlan p{};
    const long M = (long)Nb * Ho * Wo;
    const int Ktot = R * S * Cin_p;
    WgTileGeom t;
    if (pick_wgrad_tile(Nb, Hi, Wi, Cin_p, Ho, Wo, Cout, R, S, stride, pad, t)) {
        p.tile = 1;
        p.oh = t.OH;
        p.imgs = t.IMGS;
        p.splits = (int)(M / t.TP);
        p.pix_per_split = t.TP;
        p.part_floats = (long)p.splits * Cout * Ktot;
        return p;
    }

    p.tm = Cout <= 16 ? 1 : (Cout <= 32 ? 2 : 4);
    p.tn = 4;
    const long tiles = (long)((Cout + 16 * p.tm - 1) / (16 * p.tm)) * ((Ktot + 16 * p.tn - 1) / (16 * p.tn));
    // about 512 workgroups per pass, each over at least 512 output pixels
    long splits = (512 + tiles - 1) / tiles;
    const long max_splits = (M + 511) / 512;
    if (splits > max_splits) splits = max_splits;
    if (splits < 1) splits = 1;
    long pps = (M + splits - 1) / splits;
    pps = (pps + 63) / 64 * 64;
    p.pix_per_split = (int)pps;
    p.splits = (int)((M + pps - 1) / pps);
    p.part_floats = (long)p.splits * Cout * Ktot;
    return p;
}

template <int TM, int TN>
static hipError_t launch_wg(const float* dY, const float* X, float* part, const WgArgs& a, const WgradPlan& p,
                            hipStream_t st) {
    const int Ktot = a.R * a.S * a.Cin_p;
    dim3 grid((unsigned)((a.Cout + TM * 16 - 1) / (TM * 16)), (unsigned)((Ktot + TN * 16 - 1) / (TN * 16)),
              (unsigned)p.splits);
    launch((conv_wgrad_f32<TM, TN>), grid, dim3(256), 0, st, dY, X, part, a);
    return hipGetLastError();
}

template <int RS, int NG, int ST, bool K1>
static hipError_t launch_wg_tile(const float* dY, const float* X, float* part, const WgArgs& a, const WgTileGeom& t,
                                 const float* in_ss, hipStream_t st) {
    const long M = (long)a.Nb * a.Ho * a.Wo;
    dim3 grid((unsigned)(M / t.TP), (unsigned)(a.Cout / 16), (unsigned)(a.Cin_p / 16));
    const size_t lds = sizeof(float) * std::max<size_t>(((size_t)t.IMGS * t.IH * t.IW + t.TP) * 20, (size_t)4 * RS * 256);
    launch((conv_wgrad_tile_f32<RS, NG, ST, K1>), grid, dim3(256), lds, st, dY, X, part, a, t, in_ss);
    return hipGetLastError();
}

template <int RS, int ST, bool K1>
static hipError_t launch_wg_tile_ng(const float* dY, const float* X, float* part, const WgArgs& a,
                                    const WgTileGeom& t, const float* in_ss, hipStream_t st) {
    const int ng = t.TP / 64;
    if (ng == 4) return launch_wg_tile<RS, 4, ST, K1>(dY, X, part, a, t, in_ss, st);
    if (ng == 2) return launch_wg_tile<RS, 2, ST, K1>(dY, X, part, a, t, in_ss, st);
    return launch_wg_tile<RS, 1, ST, K1>(dY, X, part, a, t, in_ss, st);
}

hipError_t launch_conv_wgrad(const float* dY, const float* X, float* part, int Nb, int Hi, int Wi, int Cin_p,
                             int Ho, int Wo, int Cout, int R, int S, int stride, int pad, const WgradPlan& p,
                             hipStream_t st, const float* in_ss) {
    WgArgs a{Nb, Hi, Wi, Cin_p, Ho, Wo, Cout, R, S, stride, pad, p.pix_per_split};
    if (in_ss && !p.tile) return hipErrorInvalidValue;   // folding needs the spatial kernel
    if (p.tile) {
        WgTileGeom t;
        if (!pick_wgrad_tile(Nb, Hi, Wi, Cin_p, Ho, Wo, Cout, R, S, stride, pad, t) || t.OH != p.oh ||
            t.IMGS != p.imgs)
            return hipErrorInvalidValue;
        if (R == 1) {
            if (stride == 1) return launch_wg_tile_ng<1, 1, true>(dY, X, part, a, t, in_ss, st);
            return launch_wg_tile_ng<1, 2, true>(dY, X, part, a, t, in_ss, st);
        }
        if (stride == 1) return launch_wg_tile_ng<9, 1, false>(dY, X, part, a, t, in_ss, st);
        return launch_wg_tile_ng<9, 2, false>(dY, X, part, a, t, in_ss, st);
    }
    if (p.tm == 1) return launch_wg<1, 4>(dY, X, part, a, p, st);
    if (p.tm == 2) return launch_wg<2, 4>(dY, X, part, a, p, st);
    return launch_wg<4, 4>(dY, X, part, a, p, st);
}

// Workgroup of 1024 threads on one job: L split lanes x Q = 1024 / L output
// quads.  Thread (l, q) adds the float4 partials of quad q over splits
// l, l + L, ... (eight loads issued ahead of their adds, which stay in split
// order); the L lane sums are then halved pairwise in LDS (lane i += lane
// i + h for h = L/2, L/4, ..., 1).  A wave reads 64 / min(Q, 64) runs of
// min(Q, 64) consecutive quads of one split.
__global__ __launch_bounds__(1024) void wgrad_reduce_multi_k(const WgRedTable t) {
    __shared__ f4 red[1024];
    int j = 0;
    while (j + 1 < t.n && (int)blockIdx.x >= t.job[j + 1].wg0) ++j;
    const WgRedJob& J = t.job[j];
    const int lg = J.lanes_log2, L = 1 << lg, Q = 1024 >> lg;
    const int tid = threadIdx.x, sl = tid >> (10 - lg), qi = tid & (Q - 1);
    const long nq = (long)J.Cout * J.Ktot / 4;
    const long quad = (long)(blockIdx.x - J.wg0) * Q + qi;
    f4 s = f4{0.f, 0.f, 0.f, 0.f};
    if (quad < nq) {
        const f4* p = (const f4*)J.part + quad;
        int k = sl;
        for (; k + 7 * L < J.splits; k += 8 * L) {
            f4 v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) v[u] = p[(long)(k + u * L) * nq];
#pragma unroll
            for (int u = 0; u < 8; ++u) s += v[u];
        }
        for (; k < J.splits; k += L) s += p[(long)k * nq];
    }
    red[tid] = s;
    __syncthreads();
    for (int h = L >> 1; h > 0; h >>= 1) {
        if (sl < h) red[tid] = red[tid] + red[tid + h * Q];
        __syncthreads();
    }
    if (sl != 0 || quad >= nq) return;
    const f4 v = red[qi];
    const int co = (int)(quad * 4 / J.Ktot);
    const int col0 = (int)(quad * 4 - (long)co * J.Ktot);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const int col = col0 + e, tap = col / J.Cin_p, c = col - tap * J.Cin_p;
        if (c < J.Cin) J.g[((long)co * J.Cin + c) * J.RS + tap] = v[e];
    }
}

bool wgred_add(WgRedTable& t, const float* part, int splits, int Cout, int Ktot, int Cin, int Cin_p, int R, int S,
               float* g) {
    if (t.n >= kWgRedMaxJobs || Ktot % 4 || Ktot != R * S * Cin_p || splits < 1 ||
        ((uintptr_t)part & 15))
        return false;
    int lg = 0;
    while (lg < 6 && (8 << lg) < splits) ++lg;   // about eight splits per lane, at most 64 lanes
    const long nq = (long)Cout * Ktot / 4;
    const long wgs = (nq + (1024 >> lg) - 1) / (1024 >> lg);
    if (t.n == 0) t.wgs = 0;
    if ((long)t.wgs + wgs > 0x7fffffffL) return false;
    t.job[t.n] = WgRedJob{part, g, splits, Cout, Ktot, Cin, Cin_p, R * S, lg, t.wgs};
    t.wgs += (int)wgs;
    ++t.n;
    return true;
}

hipError_t launch_wgrad_reduce_multi(const WgRedTable& t, hipStream_t st) {
    if (t.n == 0) return hipSuccess;
    launch(wgrad_reduce_multi_k, dim3((unsigned)t.wgs), dim3(1024), 0, st, t);
    return hipGetLastError();
}

}  // namespace lpp
