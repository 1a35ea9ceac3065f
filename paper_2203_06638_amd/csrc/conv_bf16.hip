// conv_bf16.hip -- convolution passes with bfloat16 activations and weights on
// gfx950 matrix cores (v_mfma_f32_16x16x32_bf16), float32 accumulation.
//
// Forward and data-gradient passes are one implicit GEMM
//     Y[m][n] = sum_k A[m][k] * B[n][k]
// with m a pixel of the pass's output grid, n an output channel and k = (tap,
// c) a filter tap and a source channel.  A is gathered from the NHWC bf16
// source; B rows are the snapshot's bf16 weight layouts, [n][r][s][c] with c
// contiguous (W_f[cout][r][s][cin] forward, W_d[cin][r][s][cout] for the
// data gradient).  A pass is described by its taps: output pixel (i, j) reads
// source pixel (i*ss + dh, j*ss + dw) through weight tap (r, s), with
//   forward                 dh = r - pad,            ss = stride
//   data gradient, stride 1  dh = pad - r,            ss = 1
//   data gradient, stride 2  one pass per output parity class (a, b): the dX
//                            pixels (2i + a, 2j + b) receive only the taps
//                            with a + pad - r and b + pad - s even, from dY
//                            pixel (i + (a + pad - r)/2, j + (b + pad - s)/2)
// (likewise for columns), so no multiply is spent on taps between strides.
//
// Lane layout of v_mfma_f32_16x16x32_bf16 (64 lanes): lane l supplies
// A[row l%16][k = 8*(l/16) .. +8] and B[col l%16][same k] and receives
// D[rows 4*(l/16) .. +4][col l%16].  A load step is 32 values of k: four
// 8-channel chunks, each from one tap (a tap holds Cs/8 chunks; for Cs < 32 a
// step spans several taps).  Operand tiles go through LDS in rows of 32 bf16
// (64 bytes) whose four 16-byte chunks are XOR-swizzled by (row / 4) % 4, so
// both the row-wise stores and the 16-row fragment reads of 16 lanes hit
// distinct banks.  Sources of 32k channels load their tiles straight into
// LDS through a pipeline of several buffers (see the DMA notes below); the
// 8/16-channel stem stages them through registers into two buffers, the next
// step's loads in flight during the current step's MFMAs.
//
// Weight gradient: dW[cout][(tap, c)] = sum over output pixels p of
// dY[p][cout] * X[src(p, tap)][c]: a GEMM whose reduction runs over pixels.
// Both operands are pixel-major in memory, so each K-step of 32 pixels is
// written into LDS transposed (pairs of pixels packed into 32-bit words),
// after which the MFMA fragments are read exactly as in the forward kernel.
// Pixel ranges (splits) write float32 partials that a second kernel sums in
// a fixed order; nothing here uses atomics except the batch-norm sums of the
// forward epilogue in async mode (bnacc.h).
#include <algorithm>
#include <type_traits>

#include "act.h"
#include "bnacc.h"
#include "kernels.h"
#include "launch.h"

namespace lpp {

typedef __bf16 bf8 __attribute__((ext_vector_type(8)));

constexpr int kBfPitch = 32;   // forward / data-gradient operand rows (swizzled)
constexpr int kWgPitch = 40;   // weight-gradient operand rows (80 bytes, padded)

// LDS position of 16-byte chunk c (0..3) of operand row `row`
__device__ __forceinline__ int bf_swz(int c, int row) { return c ^ ((row >> 2) & 3); }

__device__ __forceinline__ f4 mfma_bf16(bf8 a, bf8 b, f4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Division of pixel indices by a grid dimension d without 64-bit or
// iterative arithmetic: n / d == umulhi(n, ceil(2^32 / d)) exactly when n * d
// < 2^32, which the launchers check for every index a kernel divides
// (largest pixel index times the divisor); magic 0 means d == 1.
__host__ __device__ inline unsigned bf_magic(unsigned d) {
    return d <= 1 ? 0u : (unsigned)((0x100000000ull + d - 1) / d);
}
__device__ __forceinline__ unsigned bf_div(unsigned n, unsigned magic) { return magic ? __umulhi(n, magic) : n; }
static inline bool bf_div_exact(long nmax, long d) { return d >= 1 && nmax >= 0 && (nmax + 1) * d <= 0x100000000L; }

// One pass of the implicit GEMM (see the header comment).
struct BfPass {
    int Hv, Wv;              // output grid of the pass
    int os, oa, ob;          // destination pixel (i*os + oa, j*os + ob)
    int Hd, Wd;              // destination tensor grid
    int ss;                  // source stride
    int nr, ns, r0, s0, step;// taps r = r0 + step*x (x < nr), s = s0 + step*y (y < ns)
    int offh, offw, sgn, shift;  // dh = (offh + sgn*r) >> shift, dw = (offw + sgn*s) >> shift
    unsigned mWv, mHv;       // bf_magic(Wv), bf_magic(Hv)
};

// Up to four passes of one launch (the parity classes of a stride-2 data
// gradient), pass blockIdx.z; a pass's workgroups beyond its grid exit.
struct BfPasses { BfPass p[4]; };

// Output channels in the epilogue: BM x BN tile, bf16, pitch BN + 8.
// FASTK (Cs % 32 == 0): a load step is 32 channels of one tap, and the tap and
// channel counters advance incrementally (no divisions in the loop);
// otherwise a step's four 8-channel chunks are decoded one by one (Cs = 8 or
// 16 spans several taps per step).  KH load steps (1 or 2) form one K-step:
// one LDS buffer, one barrier.
// res (forward only): a residual tensor of the output's shape added to the
// rounded output and rounded again, as a separate residual add of the two
// stored tensors would; the statistics then describe that sum.
// buffer resource over n bytes at p (loads past n return zeros)
__device__ __forceinline__ __amdgpu_buffer_rsrc_t bf_rsrc(const void* p, long n) {
    return __builtin_amdgcn_make_buffer_rsrc((void*)p, (short)0, (int)(n < 0x7fffffffL ? n : 0x7fffffffL), 0x00020000);
}
// 16 bytes at byte offset voff of r into LDS at dst + 16 * lane (dst uniform)
__device__ __forceinline__ void bf_dma16(__amdgpu_buffer_rsrc_t r, bf16* dst, unsigned voff) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)dst, 16, voff, 0, 0, 0);
}
// s_waitcnt immediate that waits for at most n outstanding vector memory
// operations and leaves the other counters alone
constexpr int bf_vmcnt(int n) { return (n & 15) | (7 << 4) | (15 << 8) | ((n >> 4) << 14); }
// waits until at most `ahead` K-steps of LPS loads each are in flight (ahead < NS - 1)
template <int LPS, int NS>
__device__ __forceinline__ void bf_wait_steps(int ahead) {
    static_assert(NS >= 2 && NS <= 5 && (NS - 2) * LPS < 64, "pipeline depth");
    if (NS > 4 && ahead >= 3) __builtin_amdgcn_s_waitcnt(bf_vmcnt(3 * LPS));
    else if (NS > 3 && ahead == 2) __builtin_amdgcn_s_waitcnt(bf_vmcnt(2 * LPS));
    else if (NS > 2 && ahead == 1) __builtin_amdgcn_s_waitcnt(bf_vmcnt(LPS));
    else __builtin_amdgcn_s_waitcnt(bf_vmcnt(0));
}

// DMA (FASTK only): operand tiles go from memory straight into LDS (buffer
// loads with the LDS bit: no register staging, no LDS store instructions;
// taps in the zero padding and columns past the output read out of the
// buffer's range, which yields zeros).  Each wave's load instruction fills
// 1 KB of LDS in lane order, so a thread loads the 16-byte chunk its lane
// position holds under the swizzle.  NS buffers form a pipeline: the loads
// of K-steps k+1 .. k+NS-2 are in flight while step k's fragments are read
// and its MFMAs run.  At the top of step k each thread waits (vmcnt) until at
// most the later steps' loads are outstanding -- its own loads of step k have
// then landed -- and a plain barrier (no fence, which would wait for every
// load in flight) makes everyone's landed; step k + NS - 1's loads go into
// the buffer step k - 1 used, which every wave finished reading before that
// barrier.
template <int BM, int BN, bool STATS, bool FASTK, int KH, bool DMA, int NS = 2>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(BM == 256 ? 2 : 1, 8))) void conv_bf16_k(const bf16* __restrict__ src, const bf16* __restrict__ B,
                                                   const float* __restrict__ bias, bf16* __restrict__ Y,
                                                   const bf16* __restrict__ res, ConvGeom g, BfPasses pp, int accumulate,
                                                   BnSums sums) {
    static_assert(!DMA || FASTK, "DMA operand loads need 32-channel load steps");
    static_assert(NS == 2 || DMA, "deeper pipelines use DMA operand loads");
    constexpr int TM = BM / 32, TN = BN / 32;     // 16x16 blocks per wave; waves 2 x 2
    constexpr int AL = BM / 64, BL = BN / 64;     // 16-byte operand loads per thread per K-step
    constexpr int P = kBfPitch;
    constexpr int HALF = (BM + BN) * P;           // one load step's A and B tiles
    constexpr int STAGE = KH * HALF;
    constexpr int OP = BN + 8;
    constexpr int LDSN = BM * OP > NS * STAGE ? BM * OP : NS * STAGE;   // the epilogue tile reuses the space
    // the statistics' merge area (2 x 3 x BN floats) follows, in the same
    // array: a kernel with one LDS object keeps the DMA loads' partial vmcnt
    // waits (with a second object the compiler adds a full wait before every
    // step's fragment reads)
    constexpr int REDN = STATS ? 2 * 3 * BN * 2 : 0;
    __shared__ __attribute__((aligned(16))) bf16 lds[LDSN + REDN];
    const BfPass ps = blockIdx.z == 0 ? pp.p[0] : (blockIdx.z == 1 ? pp.p[1] : (blockIdx.z == 2 ? pp.p[2] : pp.p[3]));
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave & 1, wn = wave >> 1;
    const long Mv = (long)g.Nb * ps.Hv * ps.Wv;
    const long m0 = (long)blockIdx.x * BM;
    if (m0 >= Mv) return;                         // (the whole workgroup)
    const int n0 = blockIdx.y * BN;
    const int j = tid & 3, rr = tid >> 2;
    const int RS = g.R * g.S;

    // the output rows whose A values this thread loads: the element offset of
    // the source pixel at tap offset (0, 0), and that pixel's coordinates
    int a_off[AL], a_h[AL], a_w[AL];
#pragma unroll
    for (int u = 0; u < AL; ++u) {
        const long m = m0 + rr + 64 * u;
        const bool ok = m < Mv;
        const unsigned mm = ok ? (unsigned)m : 0u;
        const unsigned t = bf_div(mm, ps.mWv);
        const int ow = (int)(mm - t * (unsigned)ps.Wv);
        const unsigned img = bf_div(t, ps.mHv);
        a_h[u] = (int)(t - img * (unsigned)ps.Hv) * ps.ss;
        a_w[u] = ow * ps.ss;
        a_off[u] = ((img * g.Hs + a_h[u]) * g.Ws + a_w[u]) * g.Cs;
        if (!ok) a_h[u] = -(1 << 20);             // every tap falls outside
    }
    const bf16* b_row[BL];
#pragma unroll
    for (int u = 0; u < BL; ++u) {
        const int n = n0 + rr + 64 * u;
        b_row[u] = n < g.Ncols ? B + (long)n * RS * g.Cs : nullptr;
    }
    const int cpt = g.Cs >> 3;                    // 8-channel chunks per tap
    const int ntap = ps.nr * ps.ns;
    const int nks = (ntap * cpt + 3) >> 2;

    uint4 ra[KH][AL], rb[KH][BL];
    // FASTK iteration state: tap (tx, ty) and the load step's first channel c0
    int tx = 0, ty = 0, c0 = 0;
    auto load_tap = [&](uint4 (&xa)[AL], uint4 (&xb)[BL], int r, int s, int ch, bool tok) {
        const int dh = (ps.offh + ps.sgn * r) >> ps.shift, dw = (ps.offw + ps.sgn * s) >> ps.shift;
        const int aoff = (dh * g.Ws + dw) * g.Cs + ch;
        const int woff = (r * g.S + s) * g.Cs + ch;
#pragma unroll
        for (int u = 0; u < AL; ++u) {
            const int h = a_h[u] + dh, w = a_w[u] + dw;
            const bool ok = tok && (unsigned)h < (unsigned)g.Hs && (unsigned)w < (unsigned)g.Ws;
            xa[u] = ok ? *(const uint4*)(src + a_off[u] + aoff) : uint4{0, 0, 0, 0};
        }
#pragma unroll
        for (int u = 0; u < BL; ++u)
            xb[u] = (tok && b_row[u]) ? *(const uint4*)(b_row[u] + woff) : uint4{0, 0, 0, 0};
    };
    // load step ks (no memory access past the last step)
    auto load = [&](uint4 (&xa)[AL], uint4 (&xb)[BL], int ks) {
        if (FASTK) {
            load_tap(xa, xb, ps.r0 + ps.step * tx, ps.s0 + ps.step * ty, c0 + 8 * j, ks < nks);
            c0 += 32;
            if (c0 == g.Cs) {
                c0 = 0;
                if (++ty == ps.ns) {
                    ty = 0;
                    ++tx;
                }
            }
        } else {
            const int kc = ks * 4 + j;
            const int tap = kc / cpt;
            const int ch = (kc - tap * cpt) * 8;
            const int x = tap / ps.ns, y = tap - (tap / ps.ns) * ps.ns;
            load_tap(xa, xb, ps.r0 + ps.step * x, ps.s0 + ps.step * y, ch, tap < ntap);
        }
    };
    auto store = [&](int buf) {
#pragma unroll
        for (int h = 0; h < KH; ++h) {
            bf16* As = lds + buf * STAGE + h * HALF;
            bf16* Bs = As + BM * P;
#pragma unroll
            for (int u = 0; u < AL; ++u) *(uint4*)(As + (rr + 64 * u) * P + bf_swz(j, rr) * 8) = ra[h][u];
#pragma unroll
            for (int u = 0; u < BL; ++u) *(uint4*)(Bs + (rr + 64 * u) * P + bf_swz(j, rr) * 8) = rb[h][u];
        }
    };
    auto load_k = [&](int kk) {
#pragma unroll
        for (int h = 0; h < KH; ++h) load(ra[h], rb[h], kk * KH + h);
    };

    f4 acc[TM][TN];
#pragma unroll
    for (int x = 0; x < TM; ++x)
#pragma unroll
        for (int y = 0; y < TN; ++y) acc[x][y] = f4{0.f, 0.f, 0.f, 0.f};

    const int nk = (nks + KH - 1) / KH;           // K-steps
    const int a_rd = ((wm * TM) * 16 + (lane & 15)) * P + bf_swz(lane >> 4, lane & 15) * 8;
    const int b_rd = BM * P + ((wn * TN) * 16 + (lane & 15)) * P + bf_swz(lane >> 4, lane & 15) * 8;
    if constexpr (DMA) {
        const __amdgpu_buffer_rsrc_t ars = bf_rsrc(src, (long)g.Nb * g.Hs * g.Ws * g.Cs * 2);
        const __amdgpu_buffer_rsrc_t brs = bf_rsrc(B, (long)g.Ncols * RS * g.Cs * 2);
        const int jj = bf_swz(j, rr);             // the source chunk of this thread's LDS position
        unsigned b_off[BL];
#pragma unroll
        for (int u = 0; u < BL; ++u) {
            const int n = n0 + rr + 64 * u;
            b_off[u] = n < g.Ncols ? (unsigned)(n * RS * g.Cs + jj * 8) * 2u : 0x80000000u;
        }
        // one K-step's loads into LDS buffer buf; (tx, ty, c0) advance
        auto issue = [&](int buf, int kk) {
#pragma unroll
            for (int h = 0; h < KH; ++h) {
                const bool tok = kk * KH + h < nks;
                const int r = ps.r0 + ps.step * tx, sc = ps.s0 + ps.step * ty;
                const int dh = (ps.offh + ps.sgn * r) >> ps.shift, dw = (ps.offw + ps.sgn * sc) >> ps.shift;
                const int aoff = (dh * g.Ws + dw) * g.Cs + c0 + jj * 8;
                const unsigned woff = (unsigned)((r * g.S + sc) * g.Cs + c0) * 2u;
                bf16* As = lds + buf * STAGE + h * HALF + wave * 16 * P;
#pragma unroll
                for (int u = 0; u < AL; ++u) {
                    const int hh = a_h[u] + dh, ww = a_w[u] + dw;
                    const bool ok = tok && (unsigned)hh < (unsigned)g.Hs && (unsigned)ww < (unsigned)g.Ws;
                    bf_dma16(ars, As + 64 * u * P, ok ? (unsigned)(a_off[u] + aoff) * 2u : 0x80000000u);
                }
#pragma unroll
                for (int u = 0; u < BL; ++u)
                    bf_dma16(brs, As + (BM + 64 * u) * P,
                             tok && b_off[u] < 0x80000000u ? b_off[u] + woff : 0x80000000u);
                c0 += 32;
                if (c0 == g.Cs) {
                    c0 = 0;
                    if (++ty == ps.ns) {
                        ty = 0;
                        ++tx;
                    }
                }
            }
        };
        constexpr int LPS = KH * (AL + BL);       // loads per K-step per thread
#pragma unroll
        for (int kk = 0; kk < NS - 1; ++kk)
            if (kk < nk) issue(kk, kk);
        int cur = 0, nxt = NS - 1;                // buffers of step kk and step kk + NS - 1
        for (int kk = 0; kk < nk; ++kk) {
            bf_wait_steps<LPS, NS>(min(NS - 2, nk - 1 - kk));
            asm volatile("s_barrier" ::: "memory");
            bf8 a[KH][TM], b[KH][TN];
#pragma unroll
            for (int h = 0; h < KH; ++h) {
                const bf16* base = lds + cur * STAGE + h * HALF;
#pragma unroll
                for (int x = 0; x < TM; ++x) a[h][x] = *(const bf8*)(base + a_rd + x * 16 * P);
#pragma unroll
                for (int y = 0; y < TN; ++y) b[h][y] = *(const bf8*)(base + b_rd + y * 16 * P);
            }
            if (kk + NS - 1 < nk) issue(nxt, kk + NS - 1);
#pragma unroll
            for (int h = 0; h < KH; ++h)
#pragma unroll
                for (int x = 0; x < TM; ++x)
#pragma unroll
                    for (int y = 0; y < TN; ++y) acc[x][y] = mfma_bf16(a[h][x], b[h][y], acc[x][y]);
            cur = cur + 1 == NS ? 0 : cur + 1;
            nxt = nxt + 1 == NS ? 0 : nxt + 1;
        }
        __syncthreads();                          // every wave is done with the buffers (the epilogue reuses them)
    } else {
    if (nk > 0) {
        load_k(0);
        store(0);
    }
    __syncthreads();
    for (int kk = 0; kk < nk; ++kk) {
        const int cur = kk & 1;
        if (kk + 1 < nk) load_k(kk + 1);
#pragma unroll
        for (int h = 0; h < KH; ++h) {
            const bf16* base = lds + cur * STAGE + h * HALF;
            bf8 a[TM], b[TN];
#pragma unroll
            for (int x = 0; x < TM; ++x) a[x] = *(const bf8*)(base + a_rd + x * 16 * P);
#pragma unroll
            for (int y = 0; y < TN; ++y) b[y] = *(const bf8*)(base + b_rd + y * 16 * P);
#pragma unroll
            for (int x = 0; x < TM; ++x)
#pragma unroll
                for (int y = 0; y < TN; ++y) acc[x][y] = mfma_bf16(a[x], b[y], acc[x][y]);
        }
        if (kk + 1 < nk) store(cur ^ 1);
        __syncthreads();
    }
    }

    // epilogue: bias, rounding to bf16 (the stored values, which the batch
    // statistics describe), transpose through LDS, 16-byte channel stores
    const int nvalid = (int)min((long)BM, Mv - m0);
    bf16* Ot = lds;
#pragma unroll
    for (int y = 0; y < TN; ++y) {
        const int col = (wn * TN + y) * 16 + (lane & 15);
        const float bb = (bias && n0 + col < g.Ncols) ? bias[n0 + col] : 0.f;
#pragma unroll
        for (int x = 0; x < TM; ++x)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int row = (wm * TM + x) * 16 + (lane >> 4) * 4 + i;
                const bf16 h = to_bf16(acc[x][y][i] + bb);
                acc[x][y][i] = from_bf16(h);
                Ot[row * OP + col] = h;
            }
    }
    __syncthreads();
    constexpr int CPR = BN / 8;                   // 16-byte chunks per tile row
    for (int e = tid; e < BM * CPR; e += 256) {
        const int row = e / CPR, ch = (e - (e / CPR) * CPR) * 8;
        const long m = m0 + row;
        if (m >= Mv || n0 + ch >= g.Ncols) continue;
        long di;
        if (ps.os == 1 && ps.Hd == ps.Hv && ps.Wd == ps.Wv) {
            di = m * g.Ncols + n0 + ch;           // the pass covers the whole output grid
        } else {
            const unsigned t = bf_div((unsigned)m, ps.mWv);
            const int ow = (int)((unsigned)m - t * (unsigned)ps.Wv);
            const unsigned img = bf_div(t, ps.mHv);
            const int oh = (int)(t - img * (unsigned)ps.Hv);
            di = ((long)((int)img * ps.Hd + oh * ps.os + ps.oa) * ps.Wd + ow * ps.os + ps.ob) * g.Ncols + n0 + ch;
        }
        bf16* dp = Y + di;
        uint4 v = *(const uint4*)(Ot + row * OP + ch);
        if (res) {
            // the residual add on the rounded values; the sum goes back into
            // the tile for the statistics
            const uint4 o = *(const uint4*)(res + di);
            const uint32_t* pv = (const uint32_t*)&v;
            const uint32_t* po = (const uint32_t*)&o;
            uint32_t w[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const float lo = __uint_as_float(pv[q] << 16) + __uint_as_float(po[q] << 16);
                const float hi = __uint_as_float(pv[q] & 0xffff0000u) + __uint_as_float(po[q] & 0xffff0000u);
                w[q] = pack_bf16x2(lo, hi);
            }
            v = uint4{w[0], w[1], w[2], w[3]};
            if (STATS) *(uint4*)(Ot + row * OP + ch) = v;
        }
        if (accumulate) {
            const uint4 o = *(const uint4*)dp;
            const uint32_t* pv = (const uint32_t*)&v;
            const uint32_t* po = (const uint32_t*)&o;
            uint32_t w[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const float lo = __uint_as_float(pv[q] << 16) + __uint_as_float(po[q] << 16);
                const float hi = __uint_as_float(pv[q] & 0xffff0000u) + __uint_as_float(po[q] & 0xffff0000u);
                w[q] = pack_bf16x2(lo, hi);
            }
            v = uint4{w[0], w[1], w[2], w[3]};
        }
        *(uint4*)dp = v;
    }
    if (STATS) {
        // per output channel of the tile: count, mean and sum of squared
        // deviations of the stored values (with a residual, the sums written
        // back into the tile)
        float(&red)[2][3][BN] = *reinterpret_cast<float(*)[2][3][BN]>(lds + LDSN);
        if (res) {
            __syncthreads();
#pragma unroll
            for (int y = 0; y < TN; ++y) {
                const int col = (wn * TN + y) * 16 + (lane & 15);
#pragma unroll
                for (int x = 0; x < TM; ++x)
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        acc[x][y][i] = from_bf16(Ot[((wm * TM + x) * 16 + (lane >> 4) * 4 + i) * OP + col]);
            }
        }
        const auto valid = [&](int x, int i) { return (wm * TM + x) * 16 + (lane >> 4) * 4 + i < nvalid; };
        const auto store = [&](int t, float n, float mu, float m2) {
            if (n0 + t < g.Ncols) tile_moments_store(sums, (int)blockIdx.x, g.Ncols, n0 + t, n, mu, m2);
        };
        if (nvalid == BM) tile_moments<TM, TN, 2, BN, true>(acc, wm, wn, valid, red, store);
        else tile_moments<TM, TN, 2, BN, false>(acc, wm, wn, valid, red, store);
    }
}

// Tile shape of a pass: BN = 128 for wide outputs, else 64; BM = 256 (one
// load step per barrier, two waves per SIMD) when that still gives `fill`
// workgroups and the source takes 32-channel load steps, else 128 when that
// does, else 64.  Measured with one stream (fill 512): the 256-row tile gains
// 10-15% where two of its workgroups fill every compute unit and loses up to
// 50% where they do not.  With four worker streams at once (fill 128) the
// larger tiles win although each pass alone is slower: WRN-16-8 +11%,
// ResNet-18 +5%, ResNet-50 +2% against fill 512 (64 and 96 are no better).
static void pick_bf16(long Mv, int Ncols, int Cs, int fill, int& bm, int& bn) {
    bn = Ncols >= 128 ? 128 : 64;
    const long nt = (Ncols + bn - 1) / bn;
    if (Cs % 32 == 0 && ((Mv + 255) / 256) * nt >= fill) {
        bm = 256;
        return;
    }
    bm = ((Mv + 127) / 128) * nt >= fill ? 128 : 64;
}

int conv_bf16_tile_rows(const ConvGeom& g) {
    int bm, bn;
    pick_bf16((long)g.Nb * g.Ho * g.Wo, g.Ncols, g.Cs, g.fill, bm, bn);
    return bm;
}

bool conv_bf16_supported(int mode, const ConvGeom& g) {
    if (g.Cs % 8 || g.Ncols % 8) return false;
    if (mode == CONV_DGRAD && g.stride != 1 && g.stride != 2) return false;
    return g.R <= 32 && g.S <= 32 && g.pad < 32;
}

template <int BM, int BN>
static hipError_t launch_bf16_pass(const bf16* src, const bf16* B, const float* bias, bf16* Y, const bf16* res,
                                   const ConvGeom& g, const BfPasses& ps, int np, bool acc, const BnSums* stats,
                                   hipStream_t st) {
    long Mmax = 0;
    for (int i = 0; i < np; ++i) Mmax = std::max(Mmax, (long)g.Nb * ps.p[i].Hv * ps.p[i].Wv);
    if (Mmax == 0) return hipSuccess;
    dim3 grid((unsigned)((Mmax + BM - 1) / BM), (unsigned)((g.Ncols + BN - 1) / BN), (unsigned)np);
    const BnSums sm = stats ? *stats : BnSums{};
    // 32-channel load steps straight into LDS, NS of them in flight; 64 x 128
    // tiles (a step of 8 MFMAs per wave) take two load steps per buffer and
    // barrier (measured 7-23% faster on 256- and 512-channel sources)
    if constexpr (BM == 64 && BN == 128) {
        if (g.Cs % 64 == 0) {
            if (stats) launch((conv_bf16_k<BM, BN, true, true, 2, true, 3>), grid, dim3(256), 0, st, src, B, bias, Y, res, g, ps, (int)acc, sm);
            else launch((conv_bf16_k<BM, BN, false, true, 2, true, 3>), grid, dim3(256), 0, st, src, B, bias, Y, res, g, ps, (int)acc, sm);
            return hipGetLastError();
        }
    }
    if (g.Cs % 32 == 0) {
        constexpr int NSD = BM == 256 ? 3 : 4;
        if (stats) launch((conv_bf16_k<BM, BN, true, true, 1, true, NSD>), grid, dim3(256), 0, st, src, B, bias, Y, res, g, ps, (int)acc, sm);
        else launch((conv_bf16_k<BM, BN, false, true, 1, true, NSD>), grid, dim3(256), 0, st, src, B, bias, Y, res, g, ps, (int)acc, sm);
    } else {
        if (stats) launch((conv_bf16_k<BM, BN, true, false, 1, false>), grid, dim3(256), 0, st, src, B, bias, Y, res, g, ps, (int)acc, sm);
        else launch((conv_bf16_k<BM, BN, false, false, 1, false>), grid, dim3(256), 0, st, src, B, bias, Y, res, g, ps, (int)acc, sm);
    }
    return hipGetLastError();
}

// np passes (1, or the four parity classes of a stride-2 data gradient) in
// one launch with tiles of bm x bn
static hipError_t run_bf16_pass(const bf16* src, const bf16* B, const float* bias, bf16* Y, const bf16* res,
                                const ConvGeom& g, const BfPasses& ps0, int np, bool acc, const BnSums* stats, int bm,
                                int bn, hipStream_t st) {
    BfPasses ps = ps0;
    for (int i = 0; i < np; ++i) {
        BfPass& q = ps.p[i];
        const long Mv = (long)g.Nb * q.Hv * q.Wv;
        if (Mv == 0) continue;                    // (its workgroups exit at once)
        // pixel indices up to Mv + BM (a tile's padding rows) divided by Wv, row indices by Hv
        if (!bf_div_exact(Mv + 256, q.Wv) || !bf_div_exact(Mv / q.Wv + 256, q.Hv)) return hipErrorInvalidValue;
        q.mWv = bf_magic((unsigned)q.Wv);
        q.mHv = bf_magic((unsigned)q.Hv);
    }
    if (bm == 256 && bn == 64) return launch_bf16_pass<256, 64>(src, B, bias, Y, res, g, ps, np, acc, stats, st);
    if (bm == 256) return launch_bf16_pass<256, 128>(src, B, bias, Y, res, g, ps, np, acc, stats, st);
    if (bm == 128 && bn == 128) return launch_bf16_pass<128, 128>(src, B, bias, Y, res, g, ps, np, acc, stats, st);
    if (bm == 128) return launch_bf16_pass<128, 64>(src, B, bias, Y, res, g, ps, np, acc, stats, st);
    if (bn == 128) return launch_bf16_pass<64, 128>(src, B, bias, Y, res, g, ps, np, acc, stats, st);
    return launch_bf16_pass<64, 64>(src, B, bias, Y, res, g, ps, np, acc, stats, st);
}

hipError_t launch_conv_bf16(int mode, const bf16* src, const bf16* B, const float* bias, bf16* Y, const ConvGeom& g,
                            bool accumulate, const BnSums* stats, hipStream_t st, const bf16* res) {
    if (!conv_bf16_supported(mode, g)) return hipErrorInvalidValue;
    if (res && (mode != CONV_FWD || accumulate)) return hipErrorInvalidValue;
    int bm, bn;
    pick_bf16((long)g.Nb * g.Ho * g.Wo, g.Ncols, g.Cs, g.fill, bm, bn);
    BfPass ps{};
    ps.Hd = g.Ho;
    ps.Wd = g.Wo;
    ps.nr = g.R;
    ps.ns = g.S;
    ps.step = 1;
    if (mode == CONV_FWD) {
        ps.Hv = g.Ho;
        ps.Wv = g.Wo;
        ps.os = 1;
        ps.ss = g.stride;
        ps.offh = ps.offw = -g.pad;
        ps.sgn = 1;
        return run_bf16_pass(src, B, bias, Y, res, g, BfPasses{{ps}}, 1, accumulate, stats, bm, bn, st);
    }
    if (stats) return hipErrorInvalidValue;
    ps.ss = 1;
    ps.sgn = -1;
    if (g.stride == 1) {
        ps.Hv = g.Ho;
        ps.Wv = g.Wo;
        ps.os = 1;
        ps.offh = ps.offw = g.pad;
        return run_bf16_pass(src, B, bias, Y, nullptr, g, BfPasses{{ps}}, 1, accumulate, nullptr, bm, bn, st);
    }
    // stride 2: one pass per parity class of the dX pixels, all four in one
    // launch, with the tile shape of the largest class
    ps.os = 2;
    ps.step = 2;
    ps.shift = 1;
    BfPasses qs{};
    long Mmax = 0;
    for (int a = 0; a < 2; ++a)
        for (int b = 0; b < 2; ++b) {
            BfPass& q = qs.p[2 * a + b];
            q = ps;
            q.oa = a;
            q.ob = b;
            q.Hv = (g.Ho - a + 1) / 2;
            q.Wv = (g.Wo - b + 1) / 2;
            q.r0 = (a + g.pad) & 1;
            q.s0 = (b + g.pad) & 1;
            q.nr = q.r0 < g.R ? (g.R - q.r0 + 1) / 2 : 0;
            q.ns = q.s0 < g.S ? (g.S - q.s0 + 1) / 2 : 0;
            q.offh = a + g.pad;
            q.offw = b + g.pad;
            Mmax = std::max(Mmax, (long)g.Nb * q.Hv * q.Wv);
        }
    int qbm, qbn;
    pick_bf16(Mmax, g.Ncols, g.Cs, g.fill, qbm, qbn);
    return run_bf16_pass(src, B, nullptr, Y, nullptr, g, qs, 4, accumulate, nullptr, qbm, qbn, st);
}

// ------------------------------------------------------------------------
// weight gradient
// ------------------------------------------------------------------------

struct WgB {
    int Nb, Hi, Wi, Cs, Ho, Wo, Cout, S, stride, pad, Ktot;
    long P;        // output pixels N*Ho*Wo
    int pps;       // pixels per split (multiple of 32)
    unsigned mWo, mHo;   // bf_magic(Wo), bf_magic(Ho)
};

// part[split][cout][col], col = (r*S + s)*Cs + c, over the split's pixels.
// Operand loads: pixel pairs (2q, 2q + 1) of the K-step, q = e & 15, with
// 8-channel chunk e >> 4 (A: output channels, B: columns).
template <int BM, int BN>
__global__ __launch_bounds__(256) void wgrad_bf16_k(const bf16* __restrict__ dY, const bf16* __restrict__ X,
                                                    float* __restrict__ part, WgB g) {
    constexpr int TM = BM / 32, TN = BN / 32;
    constexpr int P = kWgPitch;
    constexpr int STAGE = (BM + BN) * P;
    constexpr int AE = (BM * 2 + 255) / 256, BE = (BN * 2 + 255) / 256;
    __shared__ __attribute__((aligned(16))) bf16 lds[2 * STAGE];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave & 1, wn = wave >> 1;
    const int n0 = blockIdx.x * BN;               // first column
    const int m0 = blockIdx.y * BM;               // first output channel
    const long p_lo = (long)blockIdx.z * g.pps;
    const long p_hi = min(g.P, p_lo + g.pps);
    const int nks = (int)((p_hi - p_lo + 31) / 32);
    const int pq = tid & 15;

    // per load slot: A channel offset, B column tap offsets and channel
    int a_c[AE];
    bool a_ok[AE];
    int b_r[BE], b_s[BE], b_c[BE];
    bool b_ok[BE];
#pragma unroll
    for (int u = 0; u < AE; ++u) {
        const int e = tid + 256 * u;
        a_c[u] = m0 + (e >> 4) * 8;
        a_ok[u] = e < BM * 2 && a_c[u] < g.Cout;
    }
#pragma unroll
    for (int u = 0; u < BE; ++u) {
        const int e = tid + 256 * u;
        const int col = n0 + (e >> 4) * 8;
        b_ok[u] = e < BN * 2 && col < g.Ktot;
        const int tap = col / g.Cs;
        b_c[u] = col - tap * g.Cs;
        b_r[u] = tap / g.S;
        b_s[u] = tap - (tap / g.S) * g.S;
    }

    uint4 ra[AE][2], rb[BE][2];
    auto load = [&](int ks) {
        int img[2], oh[2], ow[2];
        bool pv[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const long p = p_lo + (long)ks * 32 + 2 * pq + h;
            pv[h] = p < p_hi;
            const long pp = pv[h] ? p : p_lo;
            const unsigned t = bf_div((unsigned)pp, g.mWo);
            ow[h] = (int)((unsigned)pp - t * (unsigned)g.Wo);
            const unsigned im = bf_div(t, g.mHo);
            oh[h] = (int)(t - im * (unsigned)g.Ho);
            img[h] = (int)im;
#pragma unroll
            for (int u = 0; u < AE; ++u)
                ra[u][h] = (pv[h] && a_ok[u]) ? *(const uint4*)(dY + pp * g.Cout + a_c[u]) : uint4{0, 0, 0, 0};
#pragma unroll
            for (int u = 0; u < BE; ++u) {
                const int hh = oh[h] * g.stride - g.pad + b_r[u], ww = ow[h] * g.stride - g.pad + b_s[u];
                const bool ok = pv[h] && b_ok[u] && hh >= 0 && hh < g.Hi && ww >= 0 && ww < g.Wi;
                rb[u][h] = ok ? *(const uint4*)(X + ((long)(img[h] * g.Hi + hh) * g.Wi + ww) * g.Cs + b_c[u])
                              : uint4{0, 0, 0, 0};
            }
        }
    };
    // element i of an 8-channel chunk of pixels (2q, 2q+1) -> one 32-bit word
    // of row (chunk*8 + i), columns 2q, 2q+1
    auto put = [&](bf16* base, int e, const uint4& v0, const uint4& v1) {
        const uint32_t* w0 = (const uint32_t*)&v0;
        const uint32_t* w1 = (const uint32_t*)&v1;
        bf16* rowp = base + ((e >> 4) * 8) * P + 2 * pq;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const uint32_t x0 = w0[i >> 1], x1 = w1[i >> 1];
            const uint32_t word = (i & 1) ? ((x0 >> 16) | (x1 & 0xffff0000u)) : ((x0 & 0xffffu) | (x1 << 16));
            *(uint32_t*)(rowp + i * P) = word;
        }
    };
    auto store = [&](int buf) {
        bf16* As = lds + buf * STAGE;
        bf16* Bs = As + BM * P;
#pragma unroll
        for (int u = 0; u < AE; ++u)
            if (tid + 256 * u < BM * 2) put(As, tid + 256 * u, ra[u][0], ra[u][1]);
#pragma unroll
        for (int u = 0; u < BE; ++u)
            if (tid + 256 * u < BN * 2) put(Bs, tid + 256 * u, rb[u][0], rb[u][1]);
    };

    f4 acc[TM][TN];
#pragma unroll
    for (int x = 0; x < TM; ++x)
#pragma unroll
        for (int y = 0; y < TN; ++y) acc[x][y] = f4{0.f, 0.f, 0.f, 0.f};
    if (nks > 0) {
        load(0);
        store(0);
    }
    __syncthreads();
    for (int ks = 0; ks < nks; ++ks) {
        const int cur = ks & 1;
        if (ks + 1 < nks) load(ks + 1);
        const bf16* As = lds + cur * STAGE;
        const bf16* Bs = As + BM * P;
        bf8 a[TM], b[TN];
#pragma unroll
        for (int x = 0; x < TM; ++x) a[x] = *(const bf8*)(As + ((wm * TM + x) * 16 + (lane & 15)) * P + (lane >> 4) * 8);
#pragma unroll
        for (int y = 0; y < TN; ++y) b[y] = *(const bf8*)(Bs + ((wn * TN + y) * 16 + (lane & 15)) * P + (lane >> 4) * 8);
#pragma unroll
        for (int x = 0; x < TM; ++x)
#pragma unroll
            for (int y = 0; y < TN; ++y) acc[x][y] = mfma_bf16(a[x], b[y], acc[x][y]);
        if (ks + 1 < nks) store(cur ^ 1);
        __syncthreads();
    }
    float* out = part + (long)blockIdx.z * g.Cout * g.Ktot;
#pragma unroll
    for (int x = 0; x < TM; ++x)
#pragma unroll
        for (int y = 0; y < TN; ++y) {
            const int col = n0 + (wn * TN + y) * 16 + (lane & 15);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int row = m0 + (wm * TM + x) * 16 + (lane >> 4) * 4 + i;
                if (row < g.Cout && col < g.Ktot) out[(long)row * g.Ktot + col] = acc[x][y][i];
            }
        }
}

// Weight gradient on BM x 128 tiles (BM = 128 or 64 output channels) with
// both operands loaded straight into LDS as they lie in memory (pixel-major:
// a K-step is 32 pixel rows of BM output channels for A = dY and of 128
// columns (tap, channel) for B = X at that tap) and read as MFMA fragments by
// the LDS transpose read: within each 16-lane group, lane j receives element
// j % 4 of the 8-byte reads of lanes j / 4 + 4k (k = 0..3).  So when lane s
// reads the four channels c0 + 4 (s % 4) .. + 3 of pixel row p0 + s / 4, lane
// j receives channel c0 + j at pixels p0 .. p0 + 3: half of a fragment (8
// consecutive pixels of one row of A or B), the other half from rows p0 + 4
// .. p0 + 7.  The 16-byte chunks of a row are XOR-swizzled in pairs by row,
// so that the 8 rows a half-wave's reads touch (p0 .. p0 + 3 and p0 + 8 ..
// p0 + 11) hit all 64 banks once: with 16 chunks a row the pair index is
// XORed with row bits 0, 1 and 3; with 8 (128-byte rows, two rows a bank
// cycle) with bits 1 and 3.  The operand loads run through the same NS-buffer
// pipeline as the forward kernel's.
template <int W>   // chunks (8 channels) per pixel row
__device__ __forceinline__ int wg_chunk(int c, int row) {
    const int f = W >= 16 ? ((row & 3) | (((row >> 3) & 1) << 2)) : (((row >> 1) & 1) | (((row >> 3) & 1) << 1));
    return (((c >> 1) ^ f) << 1) | (c & 1);
}

typedef short s4v __attribute__((ext_vector_type(4)));
typedef short s8v __attribute__((ext_vector_type(8)));

// ds_read_b64_tr_b16 at LDS location p.  Written out because with the
// builtin the compiler waits for every DMA load in flight before the reads,
// which would empty the pipeline at every step; the pipeline's own vmcnt
// waits and barrier already order them.  The compiler does not count these reads, so the
// caller waits for them itself (lgkm_wait) before using the results.
__device__ __forceinline__ s4v lds_read_tr16(const bf16* p) {
    const unsigned a = (unsigned)(uintptr_t)(const __attribute__((address_space(3))) bf16*)p;
    s4v r;
    asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(r) : "v"(a) : "memory");
    return r;
}
// waits until this wave's LDS reads have returned; the read values are tied
// to the wait, so that no use of them (a register copy included) moves above
template <int N>
__device__ __forceinline__ void lgkm_wait(s4v (&h)[N]) {
    static_assert(N == 12 || N == 16 || N == 24, "fragment halves per step");
    if constexpr (N == 24)
        asm volatile("s_waitcnt lgkmcnt(0)"
                     : "+v"(h[0]), "+v"(h[1]), "+v"(h[2]), "+v"(h[3]), "+v"(h[4]), "+v"(h[5]), "+v"(h[6]), "+v"(h[7]),
                       "+v"(h[8]), "+v"(h[9]), "+v"(h[10]), "+v"(h[11]), "+v"(h[12]), "+v"(h[13]), "+v"(h[14]),
                       "+v"(h[15]), "+v"(h[16]), "+v"(h[17]), "+v"(h[18]), "+v"(h[19]), "+v"(h[20]), "+v"(h[21]),
                       "+v"(h[22]), "+v"(h[23]));
    else if constexpr (N == 16)
        asm volatile("s_waitcnt lgkmcnt(0)"
                     : "+v"(h[0]), "+v"(h[1]), "+v"(h[2]), "+v"(h[3]), "+v"(h[4]), "+v"(h[5]), "+v"(h[6]), "+v"(h[7]),
                       "+v"(h[8]), "+v"(h[9]), "+v"(h[10]), "+v"(h[11]), "+v"(h[12]), "+v"(h[13]), "+v"(h[14]),
                       "+v"(h[15]));
    else
        asm volatile("s_waitcnt lgkmcnt(0)"
                     : "+v"(h[0]), "+v"(h[1]), "+v"(h[2]), "+v"(h[3]), "+v"(h[4]), "+v"(h[5]), "+v"(h[6]), "+v"(h[7]),
                       "+v"(h[8]), "+v"(h[9]), "+v"(h[10]), "+v"(h[11]));
}
__device__ __forceinline__ bf8 tr_frag(s4v lo, s4v hi) {
    return __builtin_bit_cast(bf8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

template <int BM, int NS>
__global__ __launch_bounds__(256) void wgrad_tr_bf16_k(const bf16* __restrict__ dY, const bf16* __restrict__ X,
                                                       float* __restrict__ part, WgB g) {
    static_assert(BM == 256 || BM == 128 || BM == 64, "output-channel tile");
    constexpr int TM = BM / 32, TN = 4;           // 16x16 blocks per wave; waves 2 x 2
    constexpr int WA = BM / 8, WB = 16;           // chunks per pixel row of A, of B
    constexpr int UA = BM / 64;                   // A loads per thread per K-step
    constexpr int SA = 32 * BM, STEP = SA + 32 * 128;
    __shared__ __attribute__((aligned(16))) bf16 lds[NS * STEP];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave & 1, wn = wave >> 1;
    const int n0 = blockIdx.x * 128;              // first column
    const int m0 = blockIdx.y * BM;               // first output channel
    const long p_lo = (long)blockIdx.z * g.pps;
    const long p_hi = min(g.P, p_lo + g.pps);
    const int nk = (int)((p_hi - p_lo + 31) / 32);
    const __amdgpu_buffer_rsrc_t ars = bf_rsrc(dY, g.P * g.Cout * 2);
    const __amdgpu_buffer_rsrc_t brs = bf_rsrc(X, (long)g.Nb * g.Hi * g.Wi * g.Cs * 2);

    // load slots: wave-instruction u fills 1 KB of LDS, 64 / W rows of W
    // chunks; lane % W is the physical chunk, whose logical chunk (8
    // channels) is what the lane loads
    int arow[UA], a_off[UA], brow[2], b_r[2], b_s[2], b_c[2];
    bool b_ok[2];
#pragma unroll
    for (int u = 0; u < UA; ++u) {
        arow[u] = (wave * UA + u) * (64 / WA) + lane / WA;
        const int m = m0 + wg_chunk<WA>(lane % WA, arow[u]) * 8;
        a_off[u] = m < g.Cout ? m : -1;
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        brow[u] = (wave * 2 + u) * 4 + (lane >> 4);
        const int col = n0 + wg_chunk<WB>(lane & 15, brow[u]) * 8;
        b_ok[u] = col < g.Ktot;
        const int tap = b_ok[u] ? col / g.Cs : 0;
        b_c[u] = col - tap * g.Cs;
        b_r[u] = tap / g.S;
        b_s[u] = tap - b_r[u] * g.S;
    }
    auto issue = [&](int buf, int kk) {
        bf16* As = lds + buf * STEP;
        bf16* Bs = As + SA;
        const long pk = p_lo + (long)kk * 32;
#pragma unroll
        for (int u = 0; u < UA; ++u) {
            const long p = pk + arow[u];
            const bool ok = p < p_hi && a_off[u] >= 0;
            bf_dma16(ars, As + (wave * UA + u) * 512, ok ? (unsigned)(p * g.Cout + a_off[u]) * 2u : 0x80000000u);
        }
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            const long p = pk + brow[u];
            const bool pv = p < p_hi;
            const unsigned pp = pv ? (unsigned)p : 0u;
            const unsigned t = bf_div(pp, g.mWo);
            const int ow = (int)(pp - t * (unsigned)g.Wo);
            const unsigned img = bf_div(t, g.mHo);
            const int oh = (int)(t - img * (unsigned)g.Ho);
            const int hh = oh * g.stride - g.pad + b_r[u], ww = ow * g.stride - g.pad + b_s[u];
            const bool ok = pv && b_ok[u] && (unsigned)hh < (unsigned)g.Hi && (unsigned)ww < (unsigned)g.Wi;
            bf_dma16(brs, Bs + (wave * 2 + u) * 512,
                     ok ? (unsigned)((((long)img * g.Hi + hh) * g.Wi + ww) * g.Cs + b_c[u]) * 2u : 0x80000000u);
        }
    };
    // the 16-row block at channel (or column) c16 of an operand with W chunks
    // a row: this lane's two transposed reads, into h[0] and h[1]
    const int fs = lane & 15, fg = lane >> 4;
    auto frag = [&](s4v* h, const bf16* base, int c16, auto w) {
        constexpr int W = decltype(w)::value;
#pragma unroll
        for (int k = 0; k < 2; ++k) {
            const int row = 8 * fg + 4 * k + (fs >> 2);
            const int ch = c16 + 4 * (fs & 3);
            h[k] = lds_read_tr16(base + row * (8 * W) + wg_chunk<W>(ch >> 3, row) * 8 + (ch & 7));
        }
    };

    f4 acc[TM][TN];
#pragma unroll
    for (int x = 0; x < TM; ++x)
#pragma unroll
        for (int y = 0; y < TN; ++y) acc[x][y] = f4{0.f, 0.f, 0.f, 0.f};
    constexpr int LPS = UA + 2;                   // loads per K-step per thread
#pragma unroll
    for (int kk = 0; kk < NS - 1; ++kk)
        if (kk < nk) issue(kk, kk);
    int cur = 0, nxt = NS - 1;
    for (int kk = 0; kk < nk; ++kk) {
        bf_wait_steps<LPS, NS>(min(NS - 2, nk - 1 - kk));
        asm volatile("s_barrier" ::: "memory");
        const bf16* As = lds + cur * STEP;
        const bf16* Bs = As + SA;
        s4v h[2 * (TM + TN)];                     // A fragments' halves, then B's
#pragma unroll
        for (int x = 0; x < TM; ++x) frag(h + 2 * x, As, (wm * TM + x) * 16, std::integral_constant<int, WA>{});
#pragma unroll
        for (int y = 0; y < TN; ++y)
            frag(h + 2 * (TM + y), Bs, (wn * TN + y) * 16, std::integral_constant<int, WB>{});
        if (kk + NS - 1 < nk) issue(nxt, kk + NS - 1);
        lgkm_wait(h);
#pragma unroll
        for (int x = 0; x < TM; ++x)
#pragma unroll
            for (int y = 0; y < TN; ++y)
                acc[x][y] = mfma_bf16(tr_frag(h[2 * x], h[2 * x + 1]), tr_frag(h[2 * (TM + y)], h[2 * (TM + y) + 1]),
                                      acc[x][y]);
        cur = cur + 1 == NS ? 0 : cur + 1;
        nxt = nxt + 1 == NS ? 0 : nxt + 1;
    }
    float* out = part + (long)blockIdx.z * g.Cout * g.Ktot;
#pragma unroll
    for (int x = 0; x < TM; ++x)
#pragma unroll
        for (int y = 0; y < TN; ++y) {
            const int col = n0 + (wn * TN + y) * 16 + (lane & 15);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int row = m0 + (wm * TM + x) * 16 + (lane >> 4) * 4 + i;
                if (row < g.Cout && col < g.Ktot) out[(long)row * g.Ktot + col] = acc[x][y][i];
            }
        }
}

// Tiles of 128 (64 when narrower) output channels x 128 columns and pixel
// splits for about 512 workgroups per pass, each over at least 512 pixels;
// then 256-channel tiles over the same splits where those still give 256
// workgroups (fewer, larger workgroups: half the column operand's loads per
// MFMA, and room for the other worker streams' kernels).
WgradPlan wgrad_plan_bf16(int Nb, int Ho, int Wo, int Cin_p, int Cout, int R, int S) {
    WgradPlan p{};
    const long M = (long)Nb * Ho * Wo;
    const int Ktot = R * S * Cin_p;
    p.tm = Cout >= 128 ? 128 : 64;
    p.tn = Ktot >= 128 ? 128 : 64;
    const long ktiles = (Ktot + p.tn - 1) / p.tn;
    const long tiles = (long)((Cout + p.tm - 1) / p.tm) * ktiles;
    long splits = (512 + tiles - 1) / tiles;
    const long max_splits = (M + 511) / 512;
    if (splits > max_splits) splits = max_splits;
    if (splits < 1) splits = 1;
    long pps = (M + splits - 1) / splits;
    pps = (pps + 31) / 32 * 32;
    p.pix_per_split = (int)pps;
    p.splits = (int)((M + pps - 1) / pps);
    p.part_floats = (long)p.splits * Cout * Ktot;
    if (p.tn == 128 && Cout >= 256 && ((Cout + 255) / 256) * ktiles * p.splits >= 256) p.tm = 256;
    return p;
}

template <int BM, int BN>
static hipError_t launch_wg_bf16(const bf16* dY, const bf16* X, float* part, const WgB& a, int splits,
                                 hipStream_t st) {
    dim3 grid((unsigned)((a.Ktot + BN - 1) / BN), (unsigned)((a.Cout + BM - 1) / BM), (unsigned)splits);
    launch((wgrad_bf16_k<BM, BN>), grid, dim3(256), 0, st, dY, X, part, a);
    return hipGetLastError();
}

hipError_t launch_conv_wgrad_bf16(const bf16* dY, const bf16* X, float* part, int Nb, int Hi, int Wi, int Cin_p,
                                  int Ho, int Wo, int Cout, int R, int S, int stride, int pad, const WgradPlan& p,
                                  hipStream_t st) {
    if (Cin_p % 8 || Cout % 8) return hipErrorInvalidValue;
    const long P = (long)Nb * Ho * Wo;
    if (!bf_div_exact(P, Wo) || !bf_div_exact(P / Wo, Ho)) return hipErrorInvalidValue;
    const WgB a{Nb, Hi, Wi, Cin_p, Ho, Wo, Cout, S, stride, pad, R * S * Cin_p, P, p.pix_per_split,
                bf_magic((unsigned)Wo), bf_magic((unsigned)Ho)};
    // 128-column tiles: operands through LDS as they lie, when both
    // tensors' byte offsets fit the 32-bit buffer offsets
    if (p.tn == 128 && P * Cout * 2 < 0x7fffffffL && (long)Nb * Hi * Wi * Cin_p * 2 < 0x7fffffffL) {
        dim3 grid((unsigned)((a.Ktot + 127) / 128), (unsigned)((Cout + p.tm - 1) / p.tm), (unsigned)p.splits);
        if (p.tm == 256) launch((wgrad_tr_bf16_k<256, 3>), grid, dim3(256), 0, st, dY, X, part, a);
        else if (p.tm == 128) launch((wgrad_tr_bf16_k<128, 4>), grid, dim3(256), 0, st, dY, X, part, a);
        else launch((wgrad_tr_bf16_k<64, 4>), grid, dim3(256), 0, st, dY, X, part, a);
        return hipGetLastError();
    }
    // (the register-staged kernels take 128- or 64-row tiles; the partial
    // sums' layout does not depend on the tile)
    if (p.tm >= 128 && p.tn == 128) return launch_wg_bf16<128, 128>(dY, X, part, a, p.splits, st);
    if (p.tm >= 128) return launch_wg_bf16<128, 64>(dY, X, part, a, p.splits, st);
    if (p.tn == 128) return launch_wg_bf16<64, 128>(dY, X, part, a, p.splits, st);
    return launch_wg_bf16<64, 64>(dY, X, part, a, p.splits, st);
}

}  // namespace lpp
