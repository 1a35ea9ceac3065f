// runtime.cpp -- the host side of liblpp.so: model validation and layout,
// truncated-backward plans, per-worker workspaces and streams, the step and
// averaging executors, and the C ABI declared in include/lpp.h.
//
// Paper: arXiv 2203.06638 (LPP-SGD).  Alg. 1 gives the updater and averager
// loops; Sec. 3 "Block partitions" defines the blocks; Sec. 3 "Discussion on
// the Rule" gives the reason for the truncated backward pass (a partial
// gradient only needs backpropagation from the output down to its block).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <memory>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/lpp.h"
#include "kernels.h"
#include "launch.h"

namespace lpp {
LaunchTiming& launch_timing() {
    thread_local LaunchTiming t;
    return t;
}
}  // namespace lpp

namespace {

thread_local std::string g_err;

int fail(int code, const std::string& msg) {
    g_err = msg;
    return code;
}

#define HIPCHK(expr)                                                                         \
    do {                                                                                     \
        hipError_t _e = (expr);                                                              \
        if (_e != hipSuccess) return fail(LPP_EHIP, std::string(#expr) + ": " + hipGetErrorString(_e)); \
    } while (0)

struct Shape {
    int c = 0, h = 0, w = 0;
    long numel() const { return (long)c * h * w; }
};

struct Layer {
    lpp_layer L{};
    Shape in0, in1, out;
    int dt = lpp::DT_F32;         // storage type of this layer's output and its gradient
    long poff = -1, np = 0;       // canonical parameter range
    long wcount = 0;              // conv/linear weight count (before the bias)
    int cin_p = 0;                // conv: stored channels of the input
    bool pw = false;              // conv: 1x1, stride 1, no padding, output channels not a multiple of 4 --
                                  //   run as a linear layer applied to every pixel (fp32)
    int in_bn = -1;               // conv: reads relu(bn(x)) of this BN layer's input x, folded into its loads
    int gsum_y = -1;              // conv with gsum_bn: the ReLU decision is this layer's stored output > 0 (a BN +
                                  //   residual add + ReLU group) instead of the folded BN's fma(x, scale, shift) > 0
    int gsum_bn = -1;             // conv: its data gradient (the gradient at that BN + ReLU's output) also
                                  //   forms the sums of this BN's backward
    long wf_off = -1, wd_off = -1;// conv: W_f / W_d in the worker's weight buffer (elements)
    double macs = 0;              // forward multiply-adds (conv, linear)
    lpp::WgradPlan wg{};
    // workspace offsets (bytes) of this layer's output, its gradient and aux
    // data; BN: its reduction accumulators (doubles [5][kAccSlots][C]: batch
    // sums of the forward, then sums of the backward)
    size_t act = 0, dact = 0, aux = 0, acc = 0;
};

struct Plan {
    std::vector<char> run;        // backward of this layer runs (its output grad exists)
    std::vector<char> wgrad;      // parameter gradients of this layer are written
    std::vector<char> din0, din1; // gradient into input 0 / 1 is computed
    std::vector<char> acc0, acc1; // ... and accumulated onto an earlier contribution
    double flops = 0;             // backward flops (dgrad + wgrad of conv/linear)
};

// Execution groups.  A group runs one fused kernel sequence and
// materialises exactly one layer output (`out`); layers inside a group whose
// outputs feed nothing else are never stored.
enum GKind { G_CONV, G_BNACT, G_RELU, G_ADD, G_MAXPOOL, G_GAP, G_LINEAR, G_HEAD, G_CONCAT };

// ops that read a second input (in1)
inline bool two_inputs(int op) { return op == LPP_ADD || op == LPP_CONCAT; }
struct Group {
    GKind kind = G_CONV;
    int out = -1;       // the layer whose output this group stores
    int a = -1;         // G_CONV: conv; G_BNACT: first BN; G_HEAD: pool; else: the layer
    int stats_bn = -1;  // G_CONV: BN whose batch statistics the conv epilogue computes
    int bn2 = -1;       // G_BNACT: BN of the other branch of the residual add (both normalised)
    int add = -1;       // G_BNACT / G_CONV: the residual add, if any
    int res = -1;       // G_BNACT / G_CONV: the residual tensor added unnormalised, if any
    int relu = -1;      // G_BNACT: the closing ReLU, if any; G_CONV: a ReLU applied by the conv's epilogue
    int lin = -1;       // G_HEAD: the linear layer
    bool fold = false;  // G_BNACT: BN + ReLU folded into the consuming conv (nothing launched forward)
    bool rsum = false;  // G_BNACT: its backward sums come from the data gradient of conv rsum_conv
    int rsum_conv = -1;
    bool premask = false;  // G_CONV with a ReLU: the consuming concat's backward masks its output gradient
                           //   and forms its bias gradient
    int mconv_a = -1, mconv_b = -1;  // G_CONCAT: the convs whose ReLUs (their outputs are its inputs) its
                                     //   backward applies
};

struct Model {
    lpp_model_desc desc{};
    std::vector<Layer> layers;
    int dt = lpp::DT_F32;         // activation storage type (bf16 for LPP_BF16)
    int P = 0;
    long d = 0;
    std::vector<long> blo, bhi;   // block ranges 0..P
    int img_cp = 0;               // stored channels of the image
    double fwd_flops = 0;
    std::vector<Plan> plans;      // per partition 0..P
    std::vector<std::vector<int>> consumers;
    std::vector<Group> groups;    // in execution order
    std::vector<char> stored;     // layer output materialised
    std::vector<char> gstored;    // gradient at the layer output materialised (when the backward reaches it)
    std::vector<int> gbuf;        // the layer whose gradient buffer holds it
    std::vector<int> stats_from;  // BN: conv whose epilogue computes its statistics, or -1
    // workgroups a bf16 conv pass aims for: the chip's share of one of the
    // K * P worker streams that run at once, at least a quarter of 512
    int conv_fill = 512;
};

int ceil4(int c) { return (c + 3) / 4 * 4; }
int ceil8(int c) { return (c + 7) / 8 * 8; }
size_t dt_size(int dt) { return dt == lpp::DT_BF16 ? 2 : 4; }

// Validates the description and fills shapes, parameter layout, blocks and
// plans.  Returns LPP_OK or an error code with g_err set.
int build_model(const lpp_model_desc* desc, int P, Model& M) {
    if (!desc) return fail(LPP_EINVAL, "desc is NULL");
    if (P < 1 || P > 64) return fail(LPP_EINVAL, "P must be in [1, 64]");
    const lpp_model_desc& D = *desc;
    if (D.n_layers < 1 || !D.layers) return fail(LPP_EINVAL, "model has no layers");
    if (D.batch < 1 || D.in_c < 1 || D.in_h < 1 || D.in_w < 1 || D.n_classes < 1)
        return fail(LPP_EINVAL, "batch, image shape and n_classes must be positive");
    if (D.dtype != LPP_FP32 && D.dtype != LPP_BF16) return fail(LPP_EINVAL, "unknown dtype");
    if (!(D.bn_eps > 0.f) || !std::isfinite(D.bn_eps)) return fail(LPP_EINVAL, "bn_eps must be positive");
    if (!(D.momentum >= 0.f) || !std::isfinite(D.momentum) || !std::isfinite(D.weight_decay))
        return fail(LPP_EINVAL, "momentum must be >= 0 and finite; weight_decay finite");
    M.desc = D;
    M.desc.layers = nullptr;
    M.P = P;
    M.dt = D.dtype == LPP_BF16 ? lpp::DT_BF16 : lpp::DT_F32;
    const bool bf = M.dt == lpp::DT_BF16;
    M.img_cp = bf ? ceil8(D.in_c) : ceil4(D.in_c);
    const int n = D.n_layers;
    M.layers.assign(n, Layer{});
    const Shape img{D.in_c, D.in_h, D.in_w};
    long d = 0;
    int last_block = 0;
    std::vector<char> block_seen(P + 1, 0);
    std::vector<int> consumers(n, 0);
    for (int l = 0; l < n; ++l) {
        Layer& Y = M.layers[l];
        Y.L = D.layers[l];
        const lpp_layer& L = Y.L;
        char where[64];
        snprintf(where, sizeof where, "layer %d: ", l);
        if (L.in0 < -1 || L.in0 >= l) return fail(LPP_EINVAL, std::string(where) + "in0 must be -1 or an earlier layer");
        Y.in0 = L.in0 < 0 ? img : M.layers[L.in0].out;
        if (L.in0 >= 0) consumers[L.in0]++;
        if (L.in0 < 0 && L.op != LPP_CONV)
            return fail(LPP_EUNSUPPORTED, std::string(where) + "only a conv may read the image");
        Shape o = Y.in0;
        switch (L.op) {
        case LPP_CONV: {
            if (L.cin != Y.in0.c) return fail(LPP_EINVAL, std::string(where) + "cin does not match the input");
            if (L.cout < 1 || L.k < 1 || L.stride < 1 || L.pad < 0)
                return fail(LPP_EINVAL, std::string(where) + "bad conv geometry");
            o.c = L.cout;
            o.h = (Y.in0.h + 2 * L.pad - L.k) / L.stride + 1;
            o.w = (Y.in0.w + 2 * L.pad - L.k) / L.stride + 1;
            if (Y.in0.h + 2 * L.pad < L.k || Y.in0.w + 2 * L.pad < L.k || o.h < 1 || o.w < 1)
                return fail(LPP_EINVAL, std::string(where) + "conv output is empty");
            if (L.cout % 4) {
                if (bf || L.k != 1 || L.stride != 1 || L.pad != 0 || L.in0 < 0)
                    return fail(LPP_EUNSUPPORTED, std::string(where) +
                                "cout must be a multiple of 4 (except for 1x1, stride-1, unpadded fp32 convs)");
                Y.pw = true;
            }
            Y.cin_p = L.in0 < 0 ? M.img_cp : L.cin;
            if (Y.cin_p % 4) return fail(LPP_EUNSUPPORTED, std::string(where) + "cin must be a multiple of 4");
            if (bf && (Y.cin_p % 8 || L.cout % 8))
                return fail(LPP_EUNSUPPORTED, std::string(where) + "bf16 convs need cin and cout multiples of 8");
            if (bf && L.in0 >= 0 && L.stride > 2)
                return fail(LPP_EUNSUPPORTED, std::string(where) + "bf16 data gradients need stride 1 or 2");
            Y.wcount = (long)L.cout * L.cin * L.k * L.k;
            Y.np = Y.wcount + (L.bias ? L.cout : 0);
            Y.macs = (double)D.batch * o.h * o.w * L.cout * (double)L.cin * L.k * L.k;
            break;
        }
        case LPP_BN:
            if (L.cout != Y.in0.c) return fail(LPP_EINVAL, std::string(where) + "bn channels do not match the input");
            Y.np = 2L * L.cout;
            break;
        case LPP_RELU:
            break;
        case LPP_ADD:
            if (L.in1 < -1 || L.in1 >= l) return fail(LPP_EINVAL, std::string(where) + "in1 must be an earlier layer");
            if (L.in1 < 0) return fail(LPP_EUNSUPPORTED, std::string(where) + "add cannot read the image");
            Y.in1 = M.layers[L.in1].out;
            consumers[L.in1]++;
            if (Y.in1.c != Y.in0.c || Y.in1.h != Y.in0.h || Y.in1.w != Y.in0.w)
                return fail(LPP_EINVAL, std::string(where) + "add inputs differ in shape");
            break;
        case LPP_CONCAT:
            if (L.in1 < -1 || L.in1 >= l) return fail(LPP_EINVAL, std::string(where) + "in1 must be an earlier layer");
            if (L.in1 < 0) return fail(LPP_EUNSUPPORTED, std::string(where) + "concat cannot read the image");
            Y.in1 = M.layers[L.in1].out;
            consumers[L.in1]++;
            if (Y.in1.h != Y.in0.h || Y.in1.w != Y.in0.w)
                return fail(LPP_EINVAL, std::string(where) + "concat inputs differ in spatial size");
            if (Y.in1.c % 4) return fail(LPP_EUNSUPPORTED, std::string(where) + "concat channels must be multiples of 4");
            o.c = Y.in0.c + Y.in1.c;
            break;
        case LPP_MAXPOOL:
            if (L.k < 1 || L.stride < 1 || L.pad < 0 || L.pad >= L.k || L.k * L.k > 255)
                return fail(LPP_EINVAL, std::string(where) + "bad pool geometry");
            o.h = (Y.in0.h + 2 * L.pad - L.k) / L.stride + 1;
            o.w = (Y.in0.w + 2 * L.pad - L.k) / L.stride + 1;
            if (o.h < 1 || o.w < 1) return fail(LPP_EINVAL, std::string(where) + "pool output is empty");
            break;
        case LPP_GAP:
            o.h = 1;
            o.w = 1;
            break;
        case LPP_LINEAR:
            if (Y.in0.h != 1 || Y.in0.w != 1)
                return fail(LPP_EUNSUPPORTED, std::string(where) + "linear input must be 1x1 (pool first)");
            if (L.cin != Y.in0.c || L.cout < 1) return fail(LPP_EINVAL, std::string(where) + "bad linear shape");
            if (bf && (L.in0 < 0 || D.layers[L.in0].op != LPP_GAP))
                return fail(LPP_EUNSUPPORTED, std::string(where) + "with bf16 a linear layer must read a pool");
            o.c = L.cout;
            Y.wcount = (long)L.cout * L.cin;
            Y.np = Y.wcount + (L.bias ? L.cout : 0);
            Y.macs = (double)D.batch * L.cout * L.cin;
            break;
        default:
            return fail(LPP_EINVAL, std::string(where) + "unknown op");
        }
        Y.out = o;
        Y.dt = (L.op == LPP_GAP || L.op == LPP_LINEAR) ? lpp::DT_F32 : M.dt;
        // tensors whose channels are not a multiple of 4 (a pointwise conv's
        // output) may only feed ReLU, pooling and linear layers
        const bool any_c = L.op == LPP_LINEAR || L.op == LPP_GAP || L.op == LPP_RELU || L.op == LPP_MAXPOOL;
        if (o.c % 4 && !any_c && !Y.pw)
            return fail(LPP_EUNSUPPORTED, std::string(where) + "channel counts must be multiples of 4");
        if (L.in0 >= 0 && Y.in0.c % 4 && !any_c)
            return fail(LPP_EUNSUPPORTED, std::string(where) +
                        "only ReLU, pooling and linear layers may read channels that are not a multiple of 4");
        if (L.op == LPP_RELU && ((long)D.batch * o.numel()) % 4)
            return fail(LPP_EUNSUPPORTED, std::string(where) + "relu element count must be a multiple of 4");
        if ((double)D.batch * o.numel() >= 2147483647.0 || (double)D.batch * Y.in0.h * Y.in0.w * ceil4(Y.in0.c) >= 2147483647.0)
            return fail(LPP_EUNSUPPORTED, std::string(where) + "activation exceeds 2^31 elements");
        if (Y.np > 0) {
            if (L.block < 1 || L.block > P) return fail(LPP_EINVAL, std::string(where) + "block must be in [1, P]");
            if (L.block < last_block)
                return fail(LPP_EINVAL, std::string(where) + "blocks must be contiguous runs in parameter order");
            last_block = L.block;
            block_seen[L.block] = 1;
            Y.poff = d;
            d += Y.np;
        }
    }
    for (int i = 1; i <= P; ++i)
        if (!block_seen[i]) return fail(LPP_EINVAL, "every block 1..P must own parameters");
    const Layer& last = M.layers[n - 1];
    if ((last.L.op != LPP_LINEAR && last.L.op != LPP_GAP) || last.out.c != D.n_classes)
        return fail(LPP_EINVAL, "the last layer must be a linear layer or a global pool with n_classes outputs");
    for (int l = 0; l < n - 1; ++l)
        if (consumers[l] == 0) return fail(LPP_EINVAL, "every layer but the last must feed another layer");
    if (consumers[n - 1] != 0) return fail(LPP_EINVAL, "the logits layer cannot feed another layer");
    M.d = d;
    M.blo.assign(P + 1, 0);
    M.bhi.assign(P + 1, 0);
    M.blo[0] = 0;
    M.bhi[0] = d;
    for (int i = 1; i <= P; ++i) {
        long lo = -1, hi = -1;
        for (auto& Y : M.layers)
            if (Y.np > 0 && Y.L.block == i) {
                if (lo < 0) lo = Y.poff;
                hi = Y.poff + Y.np;
            }
        M.blo[i] = lo;
        M.bhi[i] = hi;
    }
    M.fwd_flops = 0;
    for (auto& Y : M.layers) M.fwd_flops += 2.0 * Y.macs;

    // truncated-backward plans
    M.plans.assign(P + 1, Plan{});
    for (int i = 0; i <= P; ++i) {
        Plan& pl = M.plans[i];
        pl.run.assign(n, 0);
        pl.wgrad.assign(n, 0);
        pl.din0.assign(n, 0);
        pl.din1.assign(n, 0);
        pl.acc0.assign(n, 0);
        pl.acc1.assign(n, 0);
        for (int l = 0; l < n; ++l) {
            const Layer& Y = M.layers[l];
            const bool inblk = Y.np > 0 && (i == 0 || Y.L.block == i);
            pl.wgrad[l] = inblk;
            pl.run[l] = inblk || (Y.L.in0 >= 0 && pl.run[Y.L.in0]) ||
                        (two_inputs(Y.L.op) && Y.L.in1 >= 0 && pl.run[Y.L.in1]);
        }
        std::vector<char> written(n, 0);
        for (int l = n - 1; l >= 0; --l) {
            if (!pl.run[l]) continue;
            const Layer& Y = M.layers[l];
            const int a = Y.L.in0;
            if (a >= 0 && pl.run[a]) {
                pl.din0[l] = 1;
                pl.acc0[l] = written[a];
                written[a] = 1;
            }
            if (two_inputs(Y.L.op)) {
                const int b = Y.L.in1;
                if (b >= 0 && pl.run[b]) {
                    pl.din1[l] = 1;
                    pl.acc1[l] = written[b];
                    written[b] = 1;
                }
            }
            if (Y.L.op == LPP_CONV || Y.L.op == LPP_LINEAR) {
                if (pl.wgrad[l]) pl.flops += 2.0 * Y.macs;
                if (pl.din0[l]) pl.flops += 2.0 * Y.macs;
            }
        }
    }
    M.consumers.assign(n, {});
    for (int l = 0; l < n; ++l) {
        const lpp_layer& L = M.layers[l].L;
        if (L.in0 >= 0) M.consumers[L.in0].push_back(l);
        if (two_inputs(L.op) && L.in1 >= 0 && L.in1 != L.in0) M.consumers[L.in1].push_back(l);
    }
    return LPP_OK;
}

// Groups the layers for execution.  fused = false gives one group per layer
// (every activation stored).  Fused patterns:
//   conv whose only consumer is a BN: the conv epilogue computes the BN's
//     batch statistics;
//   BN [-> residual add (+ tensor | + another BN's output)] [-> ReLU], each
//     link the only consumer of the previous: one elementwise pass forward,
//     one masked reduce + apply pair backward;
//   global average pool -> linear (the logits): one head kernel with the
//     softmax cross-entropy.
void build_groups(Model& M, bool fused) {
    const int n = (int)M.layers.size();
    auto op = [&](int l) { return M.layers[l].L.op; };
    auto sole = [&](int l) { return M.consumers[l].size() == 1 ? M.consumers[l][0] : -1; };
    M.groups.clear();
    M.stored.assign(n, 0);
    M.stats_from.assign(n, -1);
    std::vector<char> taken(n, 0);
    std::vector<Group> gs;
    for (int l = 0; l < n; ++l) {
        if (taken[l]) continue;
        Group g;
        const int op_l = op(l);
        if (op_l == LPP_CONV) {
            g.kind = G_CONV;
            g.a = g.out = l;
            const int c = sole(l);
            if (fused && c >= 0 && op(c) == LPP_BN) {
                g.stats_bn = c;
                M.stats_from[c] = l;
            }
        } else if (op_l == LPP_BN) {
            g.kind = G_BNACT;
            g.a = g.out = l;
            const int c = fused ? sole(l) : -1;
            if (c >= 0 && op(c) == LPP_RELU && !taken[c]) {
                g.relu = g.out = c;
            } else if (c >= 0 && op(c) == LPP_ADD && !taken[c] && M.layers[c].L.in0 != M.layers[c].L.in1) {
                const lpp_layer& A = M.layers[c].L;
                const int other = A.in0 == l ? A.in1 : A.in0;
                g.add = g.out = c;
                if (other >= 0 && op(other) == LPP_BN && sole(other) == c && !taken[other])
                    g.bn2 = other;
                else
                    g.res = other;
                const int r = sole(c);
                if (r >= 0 && op(r) == LPP_RELU && !taken[r]) g.relu = g.out = r;
            }
        } else if (op_l == LPP_GAP) {
            const int c = fused ? sole(l) : -1;
            if (c == n - 1 && op(c) == LPP_LINEAR && M.layers[l].in0.c % 4 == 0) {
                g.kind = G_HEAD;
                g.a = l;
                g.lin = g.out = c;
            } else {
                g.kind = G_GAP;
                g.a = g.out = l;
            }
        } else {
            g.kind = op_l == LPP_RELU      ? G_RELU
                     : op_l == LPP_ADD     ? G_ADD
                     : op_l == LPP_MAXPOOL ? G_MAXPOOL
                     : op_l == LPP_CONCAT  ? G_CONCAT
                                           : G_LINEAR;
            g.a = g.out = l;
        }
        for (int x : {g.a, g.bn2, g.add, g.relu, g.lin})
            if (x >= 0) taken[x] = 1;
        gs.push_back(g);
    }
    // bf16: a conv whose only consumer is a residual add of a stored tensor
    // stores the sum itself (its epilogue adds the other input), and forms
    // the batch statistics of a BN reading the sum (a pre-activation unit's
    // end feeding the next unit's first BN)
    if (fused && M.dt == lpp::DT_BF16) {
        std::vector<int> group_of(n, -1);
        for (int i = 0; i < (int)gs.size(); ++i) group_of[gs[i].out] = i;
        std::vector<char> drop(gs.size(), 0);
        for (auto& g : gs) {
            if (g.kind != G_CONV || M.layers[g.a].pw || g.stats_bn >= 0) continue;
            const int c = sole(g.a);
            if (c < 0 || op(c) != LPP_ADD || group_of[c] < 0 || gs[group_of[c]].kind != G_ADD || drop[group_of[c]])
                continue;
            const lpp_layer& A = M.layers[c].L;
            if (A.in0 == A.in1) continue;
            const int other = A.in0 == g.a ? A.in1 : A.in0;
            if (other < 0 || group_of[other] < 0) continue;       // the residual must be a stored output
            drop[group_of[c]] = 1;
            g.add = c;
            g.res = other;
            g.out = c;
            for (int b : M.consumers[c])
                if (op(b) == LPP_BN && M.layers[b].L.in0 == c && M.stats_from[b] < 0) {
                    g.stats_bn = b;
                    M.stats_from[b] = g.a;
                    break;
                }
        }
        std::vector<Group> kept;
        for (int i = 0; i < (int)gs.size(); ++i)
            if (!drop[i]) kept.push_back(gs[i]);
        gs.swap(kept);
    }
    // fp32: a conv whose only consumer is a ReLU stores max(y, 0) from its
    // epilogue (the ReLU's output; the conv's own is never stored); the
    // backward masks the ReLU's output gradient in place, which then holds
    // the conv's
    if (fused && M.dt == lpp::DT_F32) {
        std::vector<int> group_of(n, -1);
        for (int i = 0; i < (int)gs.size(); ++i) group_of[gs[i].out] = i;
        std::vector<char> drop(gs.size(), 0);
        for (auto& g : gs) {
            if (g.kind != G_CONV || g.stats_bn >= 0 || g.add >= 0) continue;
            const int r = sole(g.a);
            if (r < 0 || op(r) != LPP_RELU || group_of[r] < 0 || gs[group_of[r]].kind != G_RELU) continue;
            drop[group_of[r]] = 1;
            g.relu = g.out = r;
        }
        std::vector<Group> kept;
        for (int i = 0; i < (int)gs.size(); ++i)
            if (!drop[i]) kept.push_back(gs[i]);
        gs.swap(kept);
    }
    // fp32: a concat of two such ReLU outputs, each consumed by it alone,
    // masks both gradient slices in its own backward (one pass instead of a
    // split pass plus a masking pass per branch)
    if (fused && M.dt == lpp::DT_F32) {
        std::vector<int> group_of(n, -1);
        for (int i = 0; i < (int)gs.size(); ++i) group_of[gs[i].out] = i;
        for (auto& g : gs) {
            if (g.kind != G_CONCAT) continue;
            const int a = M.layers[g.a].L.in0, b = M.layers[g.a].L.in1;
            if (a < 0 || b < 0 || a == b || group_of[a] < 0 || group_of[b] < 0) continue;
            Group& A = gs[group_of[a]];
            Group& B = gs[group_of[b]];
            auto ok = [&](const Group& c, int out) {
                return c.kind == G_CONV && c.relu == out && !M.layers[c.a].pw && M.consumers[out].size() == 1;
            };
            if (!ok(A, a) || !ok(B, b)) continue;
            g.mconv_a = A.a;
            g.mconv_b = B.a;
            A.premask = B.premask = true;
        }
    }
    // a group runs when its last layer's inputs exist: order by output layer
    std::stable_sort(gs.begin(), gs.end(), [](const Group& x, const Group& y) { return x.out < y.out; });
    M.groups = gs;
    M.gstored.assign(M.layers.size(), 0);
    M.gbuf.resize(M.layers.size());
    for (int l = 0; l < n; ++l) M.gbuf[l] = l;
    for (auto& g : M.groups) {
        M.stored[g.out] = 1;
        M.gstored[g.out] = 1;
        if (g.kind == G_CONV && g.relu >= 0) {
            M.gstored[g.out] = 0;
            M.gstored[g.a] = 1;
            M.gbuf[g.a] = g.out;
        }
        // the pooled features, kept for the weight gradient; their gradient
        // goes straight to the pool's input
        if (g.kind == G_HEAD) M.stored[g.a] = 1;
    }
}

// BN + ReLU groups whose only consumer is an fp32 conv that the spatial
// kernels take (forward and weight gradient): the conv reads the BN's input
// and applies relu(fma(x, scale, shift)) while staging it, so the group
// launches nothing in the forward pass and its output is never stored.
void plan_folds(Model& M, int N) {
    if (M.dt != lpp::DT_F32) return;
    for (Group& G : M.groups) {
        if (G.kind != G_BNACT || G.bn2 >= 0 || G.add >= 0 || G.relu < 0) continue;
        if (M.consumers[G.out].size() != 1) continue;
        Layer& Y = M.layers[M.consumers[G.out][0]];
        if (Y.L.op != LPP_CONV || Y.pw || Y.L.in0 != G.out || Y.cin_p != Y.L.cin) continue;
        const lpp::ConvGeom g{N, Y.in0.h, Y.in0.w, Y.cin_p, Y.out.h, Y.out.w, Y.L.cout, Y.L.k, Y.L.k, Y.L.stride,
                              Y.L.pad};
        if (!lpp::conv_fold_ok(g, Y.wg)) continue;
        G.fold = true;
        Y.in_bn = G.a;
        // the conv's data gradient is the whole gradient at the group output
        // (its only consumer): its epilogue also forms the BN backward's sums
        const lpp::ConvGeom gd{N, Y.out.h, Y.out.w, Y.L.cout, Y.in0.h, Y.in0.w, Y.L.cin, Y.L.k, Y.L.k, Y.L.stride,
                               Y.L.pad};
        // (only when the conv's group runs right after this group, so that in
        // the backward nothing runs between them that reuses the partials)
        const long gi = &G - M.groups.data();
        const bool next = gi + 1 < (long)M.groups.size() && M.groups[gi + 1].kind == G_CONV &&
                          M.groups[gi + 1].a == M.consumers[G.out][0];
        if (next && lpp::conv_dgrad_sum_tiles(gd) > 0) {
            G.rsum = true;
            G.rsum_conv = M.consumers[G.out][0];
            Y.gsum_bn = G.a;
        }
    }
    // BN + residual add of a stored tensor + ReLU (a residual unit's end)
    // whose output feeds the next unit's first conv and its shortcut: the
    // conv's data gradient, which runs last among the output's consumers and
    // adds onto the shortcut's, forms the BN backward's sums with the stored
    // output's ReLU decisions (when its group runs right after this group's)
    for (size_t gi = 0; gi + 1 < M.groups.size(); ++gi) {
        Group& G = M.groups[gi];
        if (G.kind != G_BNACT || G.fold || G.rsum || G.bn2 >= 0 || G.add < 0 || G.res < 0 || G.relu < 0) continue;
        const Group& Nx = M.groups[gi + 1];
        if (Nx.kind != G_CONV || Nx.add >= 0 || Nx.relu >= 0) continue;
        Layer& Y = M.layers[Nx.a];
        if (Y.L.op != LPP_CONV || Y.pw || Y.L.in0 != G.out || Y.cin_p != Y.L.cin || Y.in_bn >= 0) continue;
        // every other consumer of the output runs its backward before this conv's
        bool later = true;
        for (int cl : M.consumers[G.out])
            if (cl != Nx.a && cl <= Nx.out) later = false;
        if (!later) continue;
        const lpp::ConvGeom gd{N, Y.out.h, Y.out.w, Y.L.cout, Y.in0.h, Y.in0.w, Y.L.cin, Y.L.k, Y.L.k, Y.L.stride,
                               Y.L.pad};
        if (lpp::conv_dgrad_sum_tiles(gd) <= 0) continue;
        G.rsum = true;
        G.rsum_conv = Nx.a;
        Y.gsum_bn = G.a;
        Y.gsum_y = G.out;
    }
}

// ------------------------------------------------------------------------

struct Timer {
    std::mutex mu;
    std::string family;           // empty = off
    struct Rec { hipEvent_t a, b; double work; };
    std::vector<Rec> recs;
    std::vector<hipEvent_t> pool;
    double ms = 0, work = 0;
    long launches = 0;
};

struct Worker {
    hipStream_t stream = nullptr;
    bool own_stream = false;
    char* ws = nullptr;
    float* v = nullptr;
    void* wbuf = nullptr;   // conv weights in the kernels' layouts, activation type
    float* g = nullptr;
    float* m = nullptr;
    float* loss = nullptr;
    void* img = nullptr;    // the step's images, NHWC, activation type
    float* ps0 = nullptr;   // per-tile partial statistics (3 arrays)
    float* ps1 = nullptr;
    float* ps2 = nullptr;
    float* wpart = nullptr;
    lpp::StepArgs* args = nullptr;          // device: this step's images, labels, lr
    std::vector<hipGraphExec_t> graphs;     // one per partition, captured on first use
    std::vector<hipGraphExec_t> tgraphs;    // the same with the step-trace timestamps
    int last_partition = -1;
};

}  // namespace

struct lpp_ctx {
    Model M;
    int K = 0, P = 0, mode = 0;
    long dpad = 0;
    float* replicas = nullptr;               // K * dpad
    std::vector<Worker> workers;
    hipStream_t avg_stream = nullptr;
    bool own_avg = false;
    lpp::SnapEntry* snap_dev = nullptr;   // snapshot work table (entries)
    int n_snap = 0;
    long snap_tiles = 0;                  // its workgroups
    double snap_bytes = 0;                // algorithmic bytes of one snapshot
    long wbuf_floats = 0;
    size_t ws_bytes = 0;
    size_t off_v = 0, off_wbuf = 0, off_g = 0, off_m = 0, off_loss = 0, off_img = 0, off_ps = 0, off_wpart = 0,
           off_args = 0, off_acc = 0;
    long n_acc = 0;                          // doubles zeroed at the start of every step
    // sequential mode merges batch-norm reductions in a fixed order (bitwise
    // reproducible); async mode through atomic accumulators
    bool fixed_order = true;
    bool graphs = true;
    long ps_floats = 0;
    long wpart_floats = 0;                   // weight-gradient partials of one reduce batch
    std::unique_ptr<std::atomic<long>[]> counters;
    Timer timer;
    int device = 0;
    // step tracing (lpp_trace_enable): device timestamps per traced step
    // [slot][4] and per averaging round [slot][4], host records of both
    unsigned long long* trace_log = nullptr;
    unsigned long long* avg_log = nullptr;
    long trace_cap = 0;
    std::atomic<long> trace_next{0}, avg_next{0};
    std::mutex trace_mu;
    std::vector<lpp_trace_step> trace_steps;
    std::vector<lpp_trace_avg> trace_avgs;

    void* act(Worker& w, int l) { return w.ws + M.layers[l].act; }
    void* dact(Worker& w, int l) { return w.ws + M.layers[l].dact; }
    // a layer input: the image (l < 0) or a stored layer output
    const void* input(Worker& w, int l) { return l < 0 ? w.img : act(w, l); }
    // the weights of conv layer Y in forward / data-gradient layout
    const void* wf(Worker& w, const Layer& Y) { return (const char*)w.wbuf + Y.wf_off * lpp_dt_size(); }
    const void* wdg(Worker& w, const Layer& Y) { return (const char*)w.wbuf + Y.wd_off * lpp_dt_size(); }
    size_t lpp_dt_size() const { return M.dt == lpp::DT_BF16 ? 2 : 4; }
    float* aux(Worker& w, int l) { return (float*)(w.ws + M.layers[l].aux); }
    double* acc_fwd(Worker& w, int l) { return (double*)(w.ws + M.layers[l].acc); }
    double* acc_bwd(Worker& w, int l) {
        return (double*)(w.ws + M.layers[l].acc) + 2L * lpp::kAccSlots * M.layers[l].out.c;
    }
};

namespace {

template <class F>
hipError_t timed_launch(lpp_ctx* c, const char* family, double work, hipStream_t st, F&& f) {
    Timer& T = c->timer;
    bool on = false;
    hipEvent_t a = nullptr, b = nullptr;
    {
        std::lock_guard<std::mutex> g(T.mu);
        if (!T.family.empty() && T.family == family) {
            on = true;
            for (hipEvent_t* e : {&a, &b}) {
                if (!T.pool.empty()) {
                    *e = T.pool.back();
                    T.pool.pop_back();
                } else if (hipEventCreate(e) != hipSuccess) {
                    on = false;
                }
            }
        }
    }
    // the events are recorded in the dispatch packets of the launcher's
    // kernels (launch.h): the interval is the kernels' own execution
    lpp::LaunchTiming& lt = lpp::launch_timing();
    if (on) lt = lpp::LaunchTiming{a, b};
    hipError_t e = f();
    if (on) {
        const bool started = lt.start == nullptr;   // a kernel took the start event
        lt = lpp::LaunchTiming{};
        std::lock_guard<std::mutex> g(T.mu);
        if (started) {
            T.recs.push_back({a, b, work});
        } else {
            T.pool.push_back(a);
            T.pool.push_back(b);
        }
    }
    return e;
}

#define LAUNCH(fam, work, st, call)                                                              \
    do {                                                                                         \
        hipError_t _e = timed_launch(c, fam, (work), (st), [&]() { return (call); });            \
        if (_e != hipSuccess) return fail(LPP_EHIP, std::string(fam) + ": " + hipGetErrorString(_e)); \
    } while (0)

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }
long align64(long x) { return (x + 63) & ~63L; }

// Floats of weight-gradient partials kept for one batched reduce launch.
constexpr long kWpartBatch = 16L << 20;

// In async mode a batch norm's coefficients come either from the prologue of
// every apply workgroup (each re-reads C x kAccSlots fp64 sums: cheap for
// narrow layers, one launch fewer) or from one coefficient kernel, when that
// re-reading would exceed this many sums per launch.
constexpr double kPrologueSums = 4.0e6;
bool use_coef_kernel(long M, int C, int nsums) {
    return (double)lpp::bn_apply_groups(M, C) * C * lpp::kAccSlots * nsums > kPrologueSums;
}

int check_worker(const lpp_ctx* c, int w) {
    if (!c) return fail(LPP_EINVAL, "ctx is NULL");
    if (w < 0 || w >= c->K * c->P) return fail(LPP_EINVAL, "worker out of range");
    return LPP_OK;
}

int sync_all(lpp_ctx* c) {
    for (auto& w : c->workers) HIPCHK(hipStreamSynchronize(w.stream));
    HIPCHK(hipStreamSynchronize(c->avg_stream));
    return LPP_OK;
}

void destroy_ctx(lpp_ctx* c) {
    if (!c) return;
    hipSetDevice(c->device);
    for (auto& w : c->workers) {
        if (w.stream) hipStreamSynchronize(w.stream);
        for (auto g : w.graphs)
            if (g) hipGraphExecDestroy(g);
        for (auto g : w.tgraphs)
            if (g) hipGraphExecDestroy(g);
        if (w.ws) hipFree(w.ws);
        if (w.own_stream && w.stream) hipStreamDestroy(w.stream);
    }
    if (c->avg_stream) hipStreamSynchronize(c->avg_stream);
    if (c->own_avg && c->avg_stream) hipStreamDestroy(c->avg_stream);
    if (c->replicas) hipFree(c->replicas);
    if (c->snap_dev) hipFree(c->snap_dev);
    if (c->trace_log) hipFree(c->trace_log);
    if (c->avg_log) hipFree(c->avg_log);
    for (auto& r : c->timer.recs) {
        hipEventDestroy(r.a);
        hipEventDestroy(r.b);
    }
    for (auto e : c->timer.pool) hipEventDestroy(e);
    delete c;
}

// Batch-norm statistics of BN layer b into its aux (mean, rstd, scale,
// shift), from the input tensor (when no conv epilogue computed them).
int bn_stats_standalone(lpp_ctx* c, Worker& w, int b) {
    Model& M = c->M;
    Layer& B = M.layers[b];
    const int N = M.desc.batch, C = B.out.c;
    const long rows = (long)N * B.in0.h * B.in0.w;
    const void* x = c->act(w, B.L.in0);
    const int dt = M.layers[B.L.in0].dt;
    const double eb = (double)dt_size(dt);
    hipStream_t st = w.stream;
    if (c->fixed_order) {
        const lpp::BnSums out{nullptr, w.ps0, w.ps1, nullptr};
        LAUNCH("bn_stats", eb * rows * C, st, lpp::launch_stats_partial(dt, x, rows, C, out, st));
        LAUNCH("bn_stats", 0.0, st,
               lpp::launch_stats_finalize(w.ps0, w.ps1, lpp::stats_tiles(rows, C), lpp::stats_rows(rows, C), rows, C,
                                          w.v + B.poff, w.v + B.poff + C, M.desc.bn_eps, c->aux(w, b), st));
    } else {
        const lpp::BnSums out{c->acc_fwd(w, b), nullptr, nullptr, nullptr};
        LAUNCH("bn_stats", eb * rows * C, st, lpp::launch_stats_partial(dt, x, rows, C, out, st));
    }
    return LPP_OK;
}

// Forward pass of worker w at its snapshot; loss and dlogits at the end.
int run_forward(lpp_ctx* c, Worker& w) {
    Model& M = c->M;
    const int N = M.desc.batch;
    hipStream_t st = w.stream;
    const int dt = M.dt;
    const bool bf = dt == lpp::DT_BF16;
    const double eb = (double)dt_size(dt);   // bytes per stored activation element
    LAUNCH("image", (4.0 + eb) * N * M.desc.in_c * M.desc.in_h * M.desc.in_w, st,
           lpp::launch_nchw_to_nhwc(dt, w.args, w.img, N, M.desc.in_c, M.desc.in_h, M.desc.in_w, M.img_cp,
                                     (double*)(w.ws + c->off_acc), c->n_acc, st));
    bool loss_done = false;
    for (const Group& G : M.groups) {
        Layer& Y = M.layers[G.a];
        const void* x0 = c->input(w, Y.L.in0);
        const long Mrows = (long)N * Y.in0.h * Y.in0.w;
        switch (G.kind) {
        case G_CONV: {
            lpp::ConvGeom g{N, Y.in0.h, Y.in0.w, Y.cin_p, Y.out.h, Y.out.w, Y.L.cout, Y.L.k, Y.L.k, Y.L.stride, Y.L.pad};
            g.fill = M.conv_fill;
            const float* bias = Y.L.bias ? w.v + Y.poff + Y.wcount : nullptr;
            // a folded BN + ReLU: read the BN's input, normalised while staged
            lpp::BnFwd ib{};
            if (Y.in_bn >= 0) {
                const Layer& Bn = M.layers[Y.in_bn];
                x0 = c->act(w, Bn.L.in0);
                ib = lpp::BnFwd{c->fixed_order ? nullptr : c->acc_fwd(w, Y.in_bn), w.v + Bn.poff,
                                w.v + Bn.poff + Bn.out.c, M.desc.bn_eps, Mrows, c->aux(w, Y.in_bn)};
            }
            lpp::BnSums sums{};
            if (G.stats_bn >= 0) sums = c->fixed_order ? lpp::BnSums{nullptr, w.ps0, w.ps1, nullptr}
                                                       : lpp::BnSums{c->acc_fwd(w, G.stats_bn), nullptr, nullptr, nullptr};
            const lpp::BnSums* sp = G.stats_bn >= 0 ? &sums : nullptr;
            if (Y.pw)
                LAUNCH("conv_fwd", 2.0 * Y.macs, st,
                       lpp::launch_linear_fwd((const float*)x0, w.v + Y.poff, bias, (float*)c->act(w, G.out), Mrows,
                                              Y.L.cin, Y.L.cout, st, G.relu >= 0));
            else if (bf)
                LAUNCH("conv_fwd", 2.0 * Y.macs, st,
                       lpp::launch_conv_bf16(lpp::CONV_FWD, (const uint16_t*)x0, (const uint16_t*)c->wf(w, Y), bias,
                                             (uint16_t*)c->act(w, G.out), g, false, sp, st,
                                             G.add >= 0 ? (const uint16_t*)c->act(w, G.res) : nullptr));
            else
                LAUNCH("conv_fwd", 2.0 * Y.macs, st,
                       lpp::launch_conv_igemm(lpp::CONV_FWD, (const float*)x0, (const float*)c->wf(w, Y), bias,
                                              (float*)c->act(w, G.out), g,
                                              G.relu >= 0 ? lpp::kStoreRelu : lpp::kStoreSet, sp, st,
                                              Y.in_bn >= 0 ? &ib : nullptr));
            if (G.stats_bn >= 0 && c->fixed_order) {
                const Layer& B = M.layers[G.stats_bn];
                const long rows = (long)N * Y.out.h * Y.out.w;
                const int R = bf ? lpp::conv_bf16_tile_rows(g) : lpp::conv_tile_rows(g);
                const int T = (int)((rows + R - 1) / R);
                LAUNCH("bn_stats", 0.0, st,
                       lpp::launch_stats_finalize(w.ps0, w.ps1, T, R, rows, Y.L.cout, w.v + B.poff,
                                                  w.v + B.poff + Y.L.cout, M.desc.bn_eps, c->aux(w, G.stats_bn), st));
            }
            break;
        }
        case G_BNACT: {
            const int C = Y.out.c;
            if (M.stats_from[G.a] < 0) {
                int rc = bn_stats_standalone(c, w, G.a);
                if (rc) return rc;
            }
            if (G.fold) break;   // the consuming conv applies it
            if (G.bn2 >= 0 && M.stats_from[G.bn2] < 0) {
                int rc = bn_stats_standalone(c, w, G.bn2);
                if (rc) return rc;
            }
            const Layer& B1 = M.layers[G.a];
            lpp::BnFwd b1{c->fixed_order ? nullptr : c->acc_fwd(w, G.a), w.v + B1.poff, w.v + B1.poff + C,
                          M.desc.bn_eps, Mrows, c->aux(w, G.a)};
            lpp::BnFwd b2{};
            if (G.bn2 >= 0) {
                const Layer& B2 = M.layers[G.bn2];
                b2 = lpp::BnFwd{c->fixed_order ? nullptr : c->acc_fwd(w, G.bn2), w.v + B2.poff, w.v + B2.poff + C,
                                M.desc.bn_eps, Mrows, c->aux(w, G.bn2)};
            }
            if (!c->fixed_order && use_coef_kernel(Mrows, C, G.bn2 >= 0 ? 4 : 2)) {
                LAUNCH("bn_act", 0.0, st, lpp::launch_bn_fwd_coef(b1, C, st));
                b1.acc = nullptr;
                if (G.bn2 >= 0) {
                    LAUNCH("bn_act", 0.0, st, lpp::launch_bn_fwd_coef(b2, C, st));
                    b2.acc = nullptr;
                }
            }
            const void* x2 = G.bn2 >= 0 ? c->act(w, M.layers[G.bn2].L.in0) : nullptr;
            const void* r = G.res >= 0 ? c->act(w, G.res) : nullptr;
            const double bytes = 2.0 * eb * Mrows * C + (r || x2 ? eb * Mrows * C : 0.0);
            LAUNCH("bn_act", bytes, st,
                   lpp::launch_bn_act(dt, x0, b1, r, x2, G.bn2 >= 0 ? &b2 : nullptr, G.relu >= 0, c->act(w, G.out),
                                      Mrows, C, st));
            break;
        }
        case G_RELU:
            LAUNCH("relu", 2.0 * eb * Mrows * Y.out.c, st,
                   lpp::launch_relu_fwd(dt, x0, c->act(w, G.a), Mrows * Y.out.c, st));
            break;
        case G_ADD:
            LAUNCH("add", 3.0 * eb * Mrows * Y.out.c, st,
                   lpp::launch_add_fwd(dt, x0, c->act(w, Y.L.in1), c->act(w, G.a), Mrows * Y.out.c, st));
            break;
        case G_CONCAT:
            LAUNCH("concat", 2.0 * eb * Mrows * Y.out.c, st,
                   lpp::launch_concat_fwd(dt, x0, Y.in0.c, c->act(w, Y.L.in1), Y.in1.c, c->act(w, G.a), Mrows, st));
            break;
        case G_MAXPOOL:
            LAUNCH("maxpool", eb * Mrows * Y.out.c, st,
                   lpp::launch_maxpool_fwd(dt, x0, c->act(w, G.a), (uint8_t*)c->aux(w, G.a), N, Y.in0.h, Y.in0.w,
                                           Y.in0.c, Y.out.h, Y.out.w, Y.L.k, Y.L.stride, Y.L.pad, st));
            break;
        case G_GAP:
            LAUNCH("gap", eb * Mrows * Y.out.c, st,
                   lpp::launch_gap_fwd(dt, x0, (float*)c->act(w, G.a), N, Y.in0.h * Y.in0.w, Y.in0.c, st));
            break;
        case G_LINEAR: {
            const float* W = w.v + Y.poff;
            const float* bias = Y.L.bias ? W + Y.wcount : nullptr;
            LAUNCH("linear", 2.0 * Y.macs, st,
                   lpp::launch_linear_fwd((const float*)x0, W, bias, (float*)c->act(w, G.a), N, Y.L.cin, Y.L.cout,
                                          st));
            break;
        }
        case G_HEAD: {
            const Layer& L = M.layers[G.lin];
            const float* W = w.v + L.poff;
            LAUNCH("head", eb * Mrows * Y.in0.c + 2.0 * L.macs, st,
                   lpp::launch_head_fwd(dt, x0, N, Y.in0.h * Y.in0.w, Y.in0.c, W, L.L.bias ? W + L.wcount : nullptr,
                                        L.L.cout, w.args, (float*)c->act(w, G.a), (float*)c->act(w, G.lin),
                                        (float*)c->dact(w, G.lin), w.loss + 1, st));
            loss_done = true;
            break;
        }
        }
    }
    if (!loss_done) {
        const int last = (int)M.layers.size() - 1;
        LAUNCH("softmax_ce", 0.0, st,
               lpp::launch_softmax_ce((const float*)c->act(w, last), w.args, (float*)c->dact(w, last), w.loss, N,
                                      M.desc.n_classes, st));
    }
    return LPP_OK;
}

// Backward pass truncated at `partition`; parameter gradients go to w.g at
// their canonical offsets.
int run_backward(lpp_ctx* c, Worker& w, int partition) {
    Model& M = c->M;
    const Plan& pl = M.plans[partition];
    const int N = M.desc.batch;
    const int dt = M.dt;
    const bool bf = dt == lpp::DT_BF16;
    const double eb = (double)dt_size(dt);
    hipStream_t st = w.stream;
    bool loss_done = false;
    // weight-gradient partials accumulate in w.wpart until one launch sums
    // them all (when the next would not fit, the table is full, and at the end)
    lpp::WgRedTable red{};
    long woff = 0;
    auto flush_reduce = [&]() -> int {
        if (red.n == 0) return LPP_OK;
        LAUNCH("wgrad_reduce", 4.0 * woff, st, lpp::launch_wgrad_reduce_multi(red, st));
        red.n = 0;
        woff = 0;
        return LPP_OK;
    };
    for (int gi = (int)M.groups.size() - 1; gi >= 0; --gi) {
        const Group& G = M.groups[gi];
        if (!pl.run[G.out]) continue;
        Layer& Y = M.layers[G.a];
        const void* x0 = c->input(w, Y.L.in0);
        void* dy = c->dact(w, G.out);
        void* dx0 = pl.din0[G.a] ? c->dact(w, Y.L.in0) : nullptr;
        const long Min = (long)N * Y.in0.h * Y.in0.w;
        switch (G.kind) {
        case G_CONV: {
            // a fused ReLU: its output gradient masked in place into the
            // conv's, with the bias gradient's column sums on the way (with
            // premask the consuming concat's backward has done both)
            const long Mo = (long)N * Y.out.h * Y.out.w;
            const bool bias_fused = G.relu >= 0 && !Y.pw && Y.L.bias && pl.wgrad[G.a];
            if (bias_fused && !G.premask) {
                LAUNCH("relu", 3.0 * eb * Mo * Y.out.c, st,
                       lpp::launch_relu_mask_colsum(dt, dy, c->act(w, G.out), Mo, Y.L.cout, w.ps0, st));
                LAUNCH("bias_grad", 0.0, st,
                       lpp::launch_sum_from_tiles(w.ps0, lpp::stats_tiles(Mo, Y.L.cout), lpp::stats_rows(Mo, Y.L.cout),
                                                  Mo, Y.L.cout, w.g + Y.poff + Y.wcount, st));
            } else if (G.relu >= 0 && !G.premask) {
                LAUNCH("relu", 3.0 * eb * Mo * Y.out.c, st,
                       lpp::launch_relu_bwd(dt, dy, c->act(w, G.out), dy, Mo * Y.out.c, false, st));
            }
            if (Y.pw) {
                if (pl.wgrad[G.a]) {
                    const int S = Y.wg.splits, O = Y.L.cout, I = Y.L.cin, O4 = ceil4(O);
                    const long pwf = align64((long)S * O * I);
                    if (red.n + 2 > lpp::kWgRedMaxJobs || woff + align64(Y.wg.part_floats) > c->wpart_floats) {
                        int rc = flush_reduce();
                        if (rc) return rc;
                    }
                    float* part = w.wpart + woff;
                    float* partb = Y.L.bias ? part + pwf : nullptr;
                    if (!lpp::wgred_add(red, part, S, O, I, I, I, 1, 1, w.g + Y.poff) ||
                        (partb && !lpp::wgred_add(red, partb, S, 1, O4, O, O4, 1, 1, w.g + Y.poff + Y.wcount)))
                        return fail(LPP_EINVAL, "weight-gradient reduce: unsupported shape");
                    woff += align64(Y.wg.part_floats);
                    LAUNCH("conv_wgrad", 2.0 * Y.macs, st,
                           lpp::launch_linear_wgrad_part((const float*)dy, (const float*)x0, part, partb, (int)Min,
                                                         I, O, st));
                }
                if (dx0)
                    LAUNCH("conv_dgrad", 2.0 * Y.macs, st,
                           lpp::launch_linear_bwd_x((const float*)dy, w.v + Y.poff, (float*)dx0, (int)Min, Y.L.cin,
                                                    Y.L.cout, pl.acc0[G.a] != 0, st));
                break;
            }
            if (pl.wgrad[G.a]) {
                const int Ktot = Y.L.k * Y.L.k * Y.cin_p;
                const long pf = align64(Y.wg.part_floats);
                if (red.n == lpp::kWgRedMaxJobs || woff + pf > c->wpart_floats) {
                    int rc = flush_reduce();
                    if (rc) return rc;
                }
                float* part = w.wpart + woff;
                if (!lpp::wgred_add(red, part, Y.wg.splits, Y.L.cout, Ktot, Y.L.cin, Y.cin_p, Y.L.k, Y.L.k,
                                    w.g + Y.poff))
                    return fail(LPP_EINVAL, "weight-gradient reduce: unsupported shape");
                woff += pf;
                if (bf)
                    LAUNCH("conv_wgrad", 2.0 * Y.macs, st,
                           lpp::launch_conv_wgrad_bf16((const uint16_t*)dy, (const uint16_t*)x0, part, N, Y.in0.h,
                                                       Y.in0.w, Y.cin_p, Y.out.h, Y.out.w, Y.L.cout, Y.L.k, Y.L.k,
                                                       Y.L.stride, Y.L.pad, Y.wg, st));
                else if (Y.in_bn >= 0)
                    // X = relu(bn(x)) of the folded BN, rebuilt while staged
                    LAUNCH("conv_wgrad", 2.0 * Y.macs, st,
                           lpp::launch_conv_wgrad((const float*)dy, (const float*)c->act(w, M.layers[Y.in_bn].L.in0),
                                                  part, N, Y.in0.h, Y.in0.w, Y.cin_p, Y.out.h, Y.out.w, Y.L.cout,
                                                  Y.L.k, Y.L.k, Y.L.stride, Y.L.pad, Y.wg, st,
                                                  c->aux(w, Y.in_bn) + 2 * Y.cin_p));
                else
                    LAUNCH("conv_wgrad", 2.0 * Y.macs, st,
                           lpp::launch_conv_wgrad((const float*)dy, (const float*)x0, part, N, Y.in0.h, Y.in0.w,
                                                  Y.cin_p, Y.out.h, Y.out.w, Y.L.cout, Y.L.k, Y.L.k, Y.L.stride,
                                                  Y.L.pad, Y.wg, st));
                if (Y.L.bias && !bias_fused) {
                    // column sums of dY, from per-tile means
                    const lpp::BnSums tiles{nullptr, w.ps0, w.ps1, nullptr};
                    LAUNCH("bias_grad", eb * Mo * Y.L.cout, st,
                           lpp::launch_stats_partial(dt, dy, Mo, Y.L.cout, tiles, st));
                    LAUNCH("bias_grad", 0.0, st,
                           lpp::launch_sum_from_tiles(w.ps0, lpp::stats_tiles(Mo, Y.L.cout), lpp::stats_rows(Mo, Y.L.cout), Mo, Y.L.cout,
                                                      w.g + Y.poff + Y.wcount, st));
                }
            }
            if (dx0) {
                lpp::ConvGeom g{N, Y.out.h, Y.out.w, Y.L.cout, Y.in0.h, Y.in0.w, Y.L.cin, Y.L.k, Y.L.k, Y.L.stride,
                                Y.L.pad};
                g.fill = M.conv_fill;
                if (bf)
                    LAUNCH("conv_dgrad", 2.0 * Y.macs, st,
                           lpp::launch_conv_bf16(lpp::CONV_DGRAD, (const uint16_t*)dy, (const uint16_t*)c->wdg(w, Y),
                                                 nullptr, (uint16_t*)dx0, g, pl.acc0[G.a] != 0, nullptr, st));
                else if (Y.gsum_bn >= 0) {
                    // dx0 is (or completes, adding onto the shortcut's) the
                    // whole gradient at a BN + ReLU group's output: the pass
                    // also forms that BN backward's sums
                    const lpp::BnSums out = c->fixed_order ? lpp::BnSums{nullptr, w.ps0, w.ps1, nullptr}
                                                           : lpp::BnSums{c->acc_bwd(w, Y.gsum_bn), nullptr, nullptr,
                                                                         nullptr};
                    const lpp::BnBwdSum bsum{(const float*)c->act(w, M.layers[Y.gsum_bn].L.in0),
                                             c->aux(w, Y.gsum_bn),
                                             Y.gsum_y >= 0 ? (const float*)c->act(w, Y.gsum_y) : nullptr};
                    LAUNCH("conv_dgrad", 2.0 * Y.macs, st,
                           lpp::launch_conv_igemm(lpp::CONV_DGRAD, (const float*)dy, (const float*)c->wdg(w, Y),
                                                  nullptr, (float*)dx0, g, pl.acc0[G.a] != 0, &out, st, nullptr,
                                                  &bsum));
                } else
                    LAUNCH("conv_dgrad", 2.0 * Y.macs, st,
                           lpp::launch_conv_igemm(lpp::CONV_DGRAD, (const float*)dy, (const float*)c->wdg(w, Y),
                                                  nullptr, (float*)dx0, g, pl.acc0[G.a] != 0, nullptr, st));
            }
            if (G.add >= 0) {
                // the fused residual add passes the same gradient to its other input
                const lpp_layer& A = M.layers[G.add].L;
                const bool want_res = A.in0 == G.res ? pl.din0[G.add] : pl.din1[G.add];
                const bool acc_res = A.in0 == G.res ? pl.acc0[G.add] : pl.acc1[G.add];
                if (want_res)
                    LAUNCH("add", 2.0 * eb * Mo * Y.out.c, st,
                           lpp::launch_copy_acc(dt, dy, c->dact(w, G.res), Mo * Y.out.c, acc_res, st));
            }
            break;
        }
        case G_BNACT: {
            const int C = Y.out.c;
            const int b2 = G.bn2;
            int rsum_tiles = 0;   // partials of the data gradient that formed the sums
            if (G.rsum) {
                const Layer& Y2 = M.layers[G.rsum_conv];
                rsum_tiles = lpp::conv_dgrad_sum_tiles(lpp::ConvGeom{N, Y2.out.h, Y2.out.w, Y2.L.cout, Y2.in0.h,
                                                                     Y2.in0.w, Y2.L.cin, Y2.L.k, Y2.L.k,
                                                                     Y2.L.stride, Y2.L.pad});
            }
            const bool want1 = pl.run[G.a] && (pl.wgrad[G.a] || pl.din0[G.a]);
            const bool want2 = b2 >= 0 && pl.run[b2] && (pl.wgrad[b2] || pl.din0[b2]);
            bool want_res = false, acc_res = false;
            if (G.res >= 0) {
                const lpp_layer& A = M.layers[G.add].L;
                want_res = A.in0 == G.res ? pl.din0[G.add] : pl.din1[G.add];
                acc_res = A.in0 == G.res ? pl.acc0[G.add] : pl.acc1[G.add];
            }
            float* ax = c->aux(w, G.a);
            float* ax2 = b2 >= 0 ? c->aux(w, b2) : nullptr;
            const Layer* Y2 = b2 >= 0 ? &M.layers[b2] : nullptr;
            // plain BN + ReLU (fp32): the ReLU decision is recomputed from the
            // BN input and its scale and shift instead of read from the output
            const bool xmask = G.relu >= 0 && G.bn2 < 0 && G.add < 0 && !bf;
            lpp::BnBwdArgs a{dy, G.relu >= 0 && !xmask ? c->act(w, G.out) : nullptr, x0, ax, ax + C,
                             want2 ? c->act(w, Y2->L.in0) : nullptr, want2 ? ax2 : nullptr,
                             want2 ? ax2 + C : nullptr, Min, C, xmask ? ax + 2 * C : nullptr};
            float* gg1 = pl.wgrad[G.a] ? w.g + Y.poff : nullptr;
            float* gb1 = pl.wgrad[G.a] ? w.g + Y.poff + C : nullptr;
            float* gg2 = want2 && pl.wgrad[b2] ? w.g + Y2->poff : nullptr;
            float* gb2 = want2 && pl.wgrad[b2] ? w.g + Y2->poff + C : nullptr;
            lpp::BnBwdCoef k{};
            if (want1 || want2) {
                const double bytes = (a.mask ? 3.0 : 2.0) * eb * Min * C + (want2 ? eb * Min * C : 0.0);
                if (c->fixed_order) {
                    const lpp::BnSums out{nullptr, w.ps0, w.ps1, w.ps2};
                    // (a folded group's sums came from the consuming conv's data gradient)
                    if (!G.rsum) LAUNCH("bn_bwd", bytes, st, lpp::launch_bn_bwd_reduce(dt, a, out, st));
                    LAUNCH("bn_bwd", 0.0, st,
                           lpp::launch_bn_bwd_finalize(w.ps0, w.ps1, w.ps2, G.rsum ? rsum_tiles : lpp::stats_tiles(Min, C), Min, C,
                                                       w.v + Y.poff, ax + C, gg1, gb1, ax + 4 * C,
                                                       want2 ? w.v + Y2->poff : nullptr, want2 ? ax2 + C : nullptr,
                                                       gg2, gb2, want2 ? ax2 + 4 * C : nullptr, st));
                    k.coef1 = ax + 4 * C;
                    k.coef2 = want2 ? ax2 + 4 * C : nullptr;
                } else {
                    const lpp::BnSums out{c->acc_bwd(w, G.a), nullptr, nullptr, nullptr};
                    if (!G.rsum) LAUNCH("bn_bwd", bytes, st, lpp::launch_bn_bwd_reduce(dt, a, out, st));
                    k = lpp::BnBwdCoef{c->acc_bwd(w, G.a), w.v + Y.poff, gg1, gb1,
                                       want2 ? w.v + Y2->poff : nullptr, gg2, gb2, nullptr, nullptr};
                    if (use_coef_kernel(Min, C, want2 ? 3 : 2)) {
                        float* cf1 = ax + 4 * C;
                        float* cf2 = want2 ? ax2 + 4 * C : nullptr;
                        LAUNCH("bn_bwd", 0.0, st, lpp::launch_bn_bwd_coef(a, k, cf1, cf2, st));
                        k = lpp::BnBwdCoef{nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, cf1, cf2};
                    }
                }
            }
            void* d1 = want1 && pl.din0[G.a] ? dx0 : nullptr;
            void* d2 = want2 && pl.din0[b2] ? c->dact(w, Y2->L.in0) : nullptr;
            void* dr = want_res ? c->dact(w, G.res) : nullptr;
            // (with atomic sums the apply kernel also writes dgamma and dbeta)
            if (d1 || d2 || dr || (k.acc && (gg1 || gb1 || gg2 || gb2))) {
                const double bytes = ((a.mask ? 2.0 : 1.0) + (d1 ? 3.0 : 0.0) + (d2 ? 3.0 : 0.0) +
                                      (dr ? (acc_res ? 2.0 : 1.0) : 0.0)) * eb * Min * C;
                LAUNCH("bn_bwd", bytes, st,
                       lpp::launch_bn_bwd_apply(dt, a, k, d1, pl.acc0[G.a] != 0, d2, want2 && pl.acc0[b2] != 0, dr,
                                                acc_res, st));
            }
            break;
        }
        case G_RELU:
            if (dx0)
                LAUNCH("relu", 3.0 * eb * Min * Y.out.c, st,
                       lpp::launch_relu_bwd(dt, dy, x0, dx0, Min * Y.out.c, pl.acc0[G.a] != 0, st));
            break;
        case G_ADD:
            if (dx0)
                LAUNCH("add", 2.0 * eb * Min * Y.out.c, st,
                       lpp::launch_copy_acc(dt, dy, dx0, Min * Y.out.c, pl.acc0[G.a] != 0, st));
            if (pl.din1[G.a])
                LAUNCH("add", 2.0 * eb * Min * Y.out.c, st,
                       lpp::launch_copy_acc(dt, dy, c->dact(w, Y.L.in1), Min * Y.out.c, pl.acc1[G.a] != 0, st));
            break;
        case G_CONCAT:
            if (G.mconv_a >= 0 && (dx0 || pl.din1[G.a])) {
                // both inputs are fused ReLU outputs: masked slices, and the
                // two convs' bias gradients from the masked column sums
                const Layer& Ca = M.layers[G.mconv_a];
                const Layer& Cb = M.layers[G.mconv_b];
                const bool ba = Ca.L.bias && pl.wgrad[G.mconv_a], bb = Cb.L.bias && pl.wgrad[G.mconv_b];
                const int C = Y.out.c, ca = Y.in0.c, cb = Y.in1.c;
                if (pl.acc0[G.a] || pl.acc1[G.a]) return fail(LPP_EINVAL, "masked concat backward: accumulating input");
                LAUNCH("relu", (1.0 + (dx0 ? 2.0 : 0.0) * ca / C + (pl.din1[G.a] ? 2.0 : 0.0) * cb / C) * eb * Min * C, st,
                       lpp::launch_concat_relu_bwd(dt, dy, c->act(w, Y.L.in0), c->act(w, Y.L.in1), dx0,
                                                   pl.din1[G.a] ? c->dact(w, Y.L.in1) : nullptr, Min, ca, cb,
                                                   (ba || bb) ? w.ps0 : nullptr, st));
                const int T = lpp::stats_tiles(Min, C), R = lpp::stats_rows(Min, C);
                if (ba)
                    LAUNCH("bias_grad", 0.0, st,
                           lpp::launch_sum_from_tiles_ld(w.ps0, C, T, R, Min, ca, w.g + Ca.poff + Ca.wcount, st));
                if (bb)
                    LAUNCH("bias_grad", 0.0, st,
                           lpp::launch_sum_from_tiles_ld(w.ps0 + ca, C, T, R, Min, cb, w.g + Cb.poff + Cb.wcount, st));
                break;
            }
            if (dx0 || pl.din1[G.a])
                LAUNCH("concat", (1.0 + (dx0 ? 1.0 : 0.0) + (pl.din1[G.a] ? 1.0 : 0.0)) * eb * Min * Y.out.c, st,
                       lpp::launch_concat_bwd(dt, dy, Min, Y.in0.c, Y.in1.c, dx0, pl.acc0[G.a] != 0,
                                              pl.din1[G.a] ? c->dact(w, Y.L.in1) : nullptr, pl.acc1[G.a] != 0, st));
            break;
        case G_MAXPOOL:
            if (dx0)
                LAUNCH("maxpool", 2.0 * eb * Min * Y.out.c, st,
                       lpp::launch_maxpool_bwd(dt, dy, (const uint8_t*)c->aux(w, G.a), dx0, N, Y.in0.h, Y.in0.w,
                                               Y.in0.c, Y.out.h, Y.out.w, Y.L.k, Y.L.stride, Y.L.pad,
                                               pl.acc0[G.a] != 0, st));
            break;
        case G_GAP:
            if (dx0)
                LAUNCH("gap", eb * Min * Y.in0.c, st,
                       lpp::launch_gap_bwd(dt, (const float*)dy, dx0, N, Y.in0.h * Y.in0.w, Y.in0.c,
                                           pl.acc0[G.a] != 0, st));
            break;
        case G_LINEAR: {
            const float* W = w.v + Y.poff;
            if (pl.wgrad[G.a])
                LAUNCH("linear", 2.0 * Y.macs, st,
                       lpp::launch_linear_bwd_w((const float*)dy, (const float*)x0, w.g + Y.poff,
                                                Y.L.bias ? w.g + Y.poff + Y.wcount : nullptr, N, Y.L.cin, Y.L.cout,
                                                st));
            if (dx0)
                LAUNCH("linear", 2.0 * Y.macs, st,
                       lpp::launch_linear_bwd_x((const float*)dy, W, (float*)dx0, N, Y.L.cin, Y.L.cout,
                                                pl.acc0[G.a] != 0, st));
            break;
        }
        case G_HEAD: {
            const Layer& L = M.layers[G.lin];
            const bool wg = pl.wgrad[G.lin];
            LAUNCH("head", wg ? 2.0 * L.macs : 0.0, st,
                   lpp::launch_head_bwd_w((const float*)dy, (const float*)c->act(w, G.a), N, L.L.cin, L.L.cout,
                                          wg ? w.g + L.poff : nullptr,
                                          wg && L.L.bias ? w.g + L.poff + L.wcount : nullptr, w.loss + 1, w.loss,
                                          st));
            loss_done = true;
            if (dx0)
                LAUNCH("head", 2.0 * L.macs + eb * Min * Y.in0.c, st,
                       lpp::launch_head_bwd_x(dt, (const float*)dy, w.v + L.poff, N, Y.in0.h * Y.in0.w, Y.in0.c,
                                              L.L.cout, dx0, pl.acc0[G.a] != 0, w.ps0, st));
            break;
        }
        }
    }
    // the batch-mean loss, where the fused head's backward did not produce it
    bool head = false;
    for (const Group& G : M.groups) head |= G.kind == G_HEAD;
    if (head && !loss_done)
        LAUNCH("head", 0.0, st,
               lpp::launch_head_bwd_w(nullptr, nullptr, N, 1, 1, nullptr, nullptr, w.loss + 1, w.loss, st));
    return flush_reduce();
}

// The device work of one updater iteration on the worker's stream: snapshot
// of the replica, forward, truncated backward, block update.  Per-step
// arguments are read from w.args.  `traced` brackets the snapshot and the
// update with timestamp kernels (their log row comes from w.args).
int enqueue_step(lpp_ctx* c, Worker& w, int worker, int partition, bool traced) {
    const int q = worker / c->P;
    float* xq = c->replicas + (long)q * c->dpad;
    hipStream_t st = w.stream;
    if (traced) HIPCHK(lpp::launch_timestamp(c->trace_log, w.args, -1, 0, st));
    LAUNCH("snapshot", c->snap_bytes, st,
           lpp::launch_snapshot(c->M.dt, xq, w.v, c->snap_dev, c->n_snap, c->snap_tiles, w.wbuf, st));
    if (traced) HIPCHK(lpp::launch_timestamp(c->trace_log, w.args, -1, 1, st));
    int rc = run_forward(c, w);
    if (rc) return rc;
    rc = run_backward(c, w, partition);
    if (rc) return rc;
    const long lo = c->M.blo[partition], hi = c->M.bhi[partition];
    const bool mom = c->M.desc.momentum != 0.f;
    if (traced) HIPCHK(lpp::launch_timestamp(c->trace_log, w.args, -1, 2, st));
    LAUNCH("sgd_update", (mom ? 20.0 : 12.0) * (hi - lo), st,
           lpp::launch_sgd_update(xq, mom ? w.m : nullptr, w.g, lo, hi, w.args, 0.f, c->M.desc.momentum,
                                  c->M.desc.weight_decay, st));
    if (traced) HIPCHK(lpp::launch_timestamp(c->trace_log, w.args, -1, 3, st));
    return LPP_OK;
}

}  // namespace

// ========================================================================
// C ABI
// ========================================================================

extern "C" {

const char* lpp_last_error(void) { return g_err.c_str(); }

int lpp_describe(const lpp_model_desc* desc, int P, lpp_model_info* out) {
    if (!out) return fail(LPP_EINVAL, "out is NULL");
    Model M;
    int rc = build_model(desc, P, M);
    if (rc) return rc;
    memset(out, 0, sizeof *out);
    out->d = M.d;
    out->P = P;
    for (int i = 0; i <= P; ++i) {
        out->block_lo[i] = M.blo[i];
        out->block_hi[i] = M.bhi[i];
        out->bwd_flops[i] = M.plans[i].flops;
    }
    out->fwd_flops = M.fwd_flops;
    return LPP_OK;
}

int lpp_init(const lpp_model_desc* desc, int K, int P, const lpp_options* opt, lpp_ctx** out) {
    if (!out) return fail(LPP_EINVAL, "out is NULL");
    *out = nullptr;
    if (K < 1 || K > lpp::kMaxReplicas) return fail(LPP_EINVAL, "K must be in [1, 16]");
    std::unique_ptr<lpp_ctx, void (*)(lpp_ctx*)> c(new lpp_ctx, destroy_ctx);
    int rc = build_model(desc, P, c->M);
    if (rc) return rc;
    c->K = K;
    c->P = P;
    c->M.conv_fill = std::max(128, 512 / (K * std::max(P, 1)));
    c->mode = opt ? opt->mode : LPP_SEQUENTIAL;
    c->fixed_order = c->mode == LPP_SEQUENTIAL;
    if (c->mode != LPP_SEQUENTIAL && c->mode != LPP_ASYNC) return fail(LPP_EINVAL, "unknown mode");
    build_groups(c->M, !(opt && opt->unfused));
    c->graphs = !(opt && opt->no_graphs);
    HIPCHK(hipGetDevice(&c->device));
    Model& M = c->M;
    const int N = M.desc.batch;
    const long d = M.d;
    c->dpad = (d + 63) / 64 * 64;

    // conv weight layouts and the snapshot table
    std::vector<lpp::SnapConvDesc> snaps;
    long wf = 0;
    for (auto& Y : M.layers) {
        if (Y.L.op == LPP_CONV && Y.pw) {
            // weight (and bias) gradient partials over row splits
            const long rows = (long)N * Y.in0.h * Y.in0.w;
            Y.wg = lpp::WgradPlan{};
            Y.wg.splits = lpp::linear_wgrad_splits(rows);
            Y.wg.part_floats = align64((long)Y.wg.splits * Y.L.cout * Y.L.cin) +
                               (Y.L.bias ? align64((long)Y.wg.splits * ceil4(Y.L.cout)) : 0);
        }
        if (Y.L.op != LPP_CONV || Y.pw) continue;
        const long nf = (long)Y.L.cout * Y.L.k * Y.L.k * Y.cin_p;
        const long nd = (long)Y.L.cin * Y.L.k * Y.L.k * Y.L.cout;
        Y.wf_off = wf;
        wf += (nf + 63) / 64 * 64;
        Y.wd_off = wf;
        wf += (nd + 63) / 64 * 64;
        snaps.push_back({Y.poff, Y.L.cout, Y.L.cin, Y.cin_p, Y.L.k, Y.L.k, Y.wf_off, Y.wd_off});
        Y.wg = M.dt == lpp::DT_BF16 ? lpp::wgrad_plan_bf16(N, Y.out.h, Y.out.w, Y.cin_p, Y.L.cout, Y.L.k, Y.L.k)
                                     : lpp::wgrad_plan(N, Y.in0.h, Y.in0.w, Y.cin_p, Y.out.h, Y.out.w, Y.L.cout,
                                                       Y.L.k, Y.L.k, Y.L.stride, Y.L.pad);
    }
    if (!(opt && opt->unfused)) plan_folds(M, N);
    c->wbuf_floats = wf;
    std::vector<lpp::SnapEntry> snap_tab(2 * snaps.size() + 1);
    c->snap_tiles = lpp::snapshot_table(snaps.data(), (int)snaps.size(), d, M.dt, snap_tab.data(),
                                        (int)snap_tab.size(), &c->n_snap, &c->snap_bytes);
    if (c->snap_tiles < 0)
        return fail(LPP_EUNSUPPORTED, "conv output channels must be multiples of 4 (8 for bf16) for the snapshot");
    snap_tab.resize(c->n_snap);

    // workspace layout (bytes)
    size_t off = 0;
    auto take = [&](size_t bytes) {
        size_t o = off;
        off = align256(off + bytes);
        return o;
    };
    c->off_v = take(sizeof(float) * c->dpad);
    const size_t eb = dt_size(M.dt);
    c->off_wbuf = take(eb * std::max<long>(wf, 1));
    c->off_g = take(sizeof(float) * c->dpad);
    c->off_m = take(sizeof(float) * c->dpad);
    c->off_loss = take(sizeof(float) * (1 + N));
    c->off_args = take(sizeof(lpp::StepArgs));
    c->off_img = take(eb * (size_t)N * M.desc.in_h * M.desc.in_w * M.img_cp);
    long ps = 1, wpart = 1, wsum = 0;
    for (int l = 0; l < (int)M.layers.size(); ++l) {
        Layer& Y = M.layers[l];
        const long rows_out = (long)N * Y.out.h * Y.out.w;
        if (M.stored[l]) {
            Y.act = take(dt_size(Y.dt) * (size_t)rows_out * Y.out.c);
            Y.dact = take(dt_size(Y.dt) * (size_t)rows_out * Y.out.c);
        }
        if (Y.L.op == LPP_BN) Y.aux = take(sizeof(float) * 7 * Y.out.c);
        if (Y.L.op == LPP_MAXPOOL) Y.aux = take((size_t)rows_out * Y.out.c);
        const long rin = (long)N * Y.in0.h * Y.in0.w;
        if (Y.L.op == LPP_BN) ps = std::max<long>(ps, (long)lpp::stats_tiles(rin, Y.out.c) * Y.out.c);
        if (Y.L.op == LPP_LINEAR) ps = std::max<long>(ps, (long)N * Y.L.cin);   // the wide head's dfeat
        if (Y.L.op == LPP_CONCAT) ps = std::max<long>(ps, (long)lpp::stats_tiles(rows_out, Y.out.c) * Y.out.c);
        if (Y.L.op == LPP_CONV && !Y.pw) {
            lpp::ConvGeom g{N, Y.in0.h, Y.in0.w, Y.cin_p, Y.out.h, Y.out.w, Y.L.cout, Y.L.k, Y.L.k, Y.L.stride,
                            Y.L.pad};
            g.fill = M.conv_fill;
            const int tr = M.dt == lpp::DT_BF16 ? lpp::conv_bf16_tile_rows(g) : lpp::conv_tile_rows(g);
            const long tiles = (rows_out + tr - 1) / tr;
            ps = std::max<long>(ps, tiles * Y.L.cout);
            ps = std::max<long>(ps, (long)lpp::stats_tiles(rows_out, Y.L.cout) * Y.L.cout);
            if (Y.gsum_bn >= 0) {
                const lpp::ConvGeom gd{N, Y.out.h, Y.out.w, Y.L.cout, Y.in0.h, Y.in0.w, Y.L.cin, Y.L.k, Y.L.k,
                                       Y.L.stride, Y.L.pad};
                ps = std::max<long>(ps, (long)lpp::conv_dgrad_sum_tiles(gd) * Y.L.cin);
            }
            wpart = std::max<long>(wpart, align64(Y.wg.part_floats));
            wsum += align64(Y.wg.part_floats);
        }
        if (Y.L.op == LPP_CONV && Y.pw) {
            wpart = std::max<long>(wpart, align64(Y.wg.part_floats));
            wsum += align64(Y.wg.part_floats);
        }
    }
    // the partials of consecutive weight gradients stay until one reduce
    // launch sums them (at most kWpartBatch floats, or one gradient's)
    wpart = std::max<long>(wpart, std::min<long>(wsum, kWpartBatch));
    c->wpart_floats = wpart;
    c->off_acc = off;
    for (Layer& Y : M.layers)
        if (Y.L.op == LPP_BN) Y.acc = take(sizeof(double) * 5 * lpp::kAccSlots * Y.out.c);
    c->n_acc = (long)((off - c->off_acc) / sizeof(double));
    c->ps_floats = ps;
    c->off_ps = take(sizeof(float) * 3 * ps);
    c->off_wpart = take(sizeof(float) * wpart);
    c->ws_bytes = off;

    // device allocations
    if (hipMalloc((void**)&c->replicas, sizeof(float) * c->dpad * K) != hipSuccess)
        return fail(LPP_ENOMEM, "replica allocation failed");
    HIPCHK(hipMemset(c->replicas, 0, sizeof(float) * c->dpad * K));
    if (!snap_tab.empty()) {
        if (hipMalloc((void**)&c->snap_dev, sizeof(lpp::SnapEntry) * snap_tab.size()) != hipSuccess)
            return fail(LPP_ENOMEM, "snapshot table allocation failed");
        HIPCHK(hipMemcpy(c->snap_dev, snap_tab.data(), sizeof(lpp::SnapEntry) * snap_tab.size(),
                         hipMemcpyHostToDevice));
    }
    c->counters.reset(new std::atomic<long>[K]);
    for (int q = 0; q < K; ++q) c->counters[q].store(0);
    c->workers.resize((size_t)K * P);
    for (int i = 0; i < K * P; ++i) {
        Worker& w = c->workers[i];
        if (opt && opt->worker_streams && opt->worker_streams[i]) {
            w.stream = (hipStream_t)opt->worker_streams[i];
        } else {
            HIPCHK(hipStreamCreateWithFlags(&w.stream, hipStreamNonBlocking));
            w.own_stream = true;
        }
        if (hipMalloc((void**)&w.ws, c->ws_bytes) != hipSuccess)
            return fail(LPP_ENOMEM, "worker workspace allocation failed");
        HIPCHK(hipMemset(w.ws, 0, c->ws_bytes));
        w.v = (float*)(w.ws + c->off_v);
        w.wbuf = w.ws + c->off_wbuf;
        w.g = (float*)(w.ws + c->off_g);
        w.m = (float*)(w.ws + c->off_m);
        w.loss = (float*)(w.ws + c->off_loss);
        w.img = w.ws + c->off_img;
        w.ps0 = (float*)(w.ws + c->off_ps);
        w.ps1 = w.ps0 + c->ps_floats;
        w.ps2 = w.ps1 + c->ps_floats;
        w.wpart = (float*)(w.ws + c->off_wpart);
        w.args = (lpp::StepArgs*)(w.ws + c->off_args);
        w.graphs.assign(P + 1, nullptr);
        w.tgraphs.assign(P + 1, nullptr);
    }
    if (opt && opt->avg_stream) {
        c->avg_stream = (hipStream_t)opt->avg_stream;
    } else {
        HIPCHK(hipStreamCreateWithFlags(&c->avg_stream, hipStreamNonBlocking));
        c->own_avg = true;
    }
    HIPCHK(hipDeviceSynchronize());
    *out = c.release();
    return LPP_OK;
}

int lpp_destroy(lpp_ctx* c) {
    if (!c) return fail(LPP_EINVAL, "ctx is NULL");
    destroy_ctx(c);
    return LPP_OK;
}

int lpp_step(lpp_ctx* c, int worker, const lpp_batch* batch, int partition, float lr) {
    int rc = check_worker(c, worker);
    if (rc) return rc;
    if (!batch || !batch->images || !batch->labels) return fail(LPP_EINVAL, "batch or its buffers are NULL");
    if (batch->n != c->M.desc.batch) return fail(LPP_EINVAL, "batch->n must equal the model's batch");
    if (partition < 0 || partition > c->P) return fail(LPP_EINVAL, "partition must be in [0, P]");
    if (!std::isfinite(lr)) return fail(LPP_EINVAL, "lr must be finite");
    Worker& w = c->workers[worker];
    const int q = worker / c->P;
    const long s_read = c->counters[q].fetch_add(1);   // s := read&inc(C^q)
    hipStream_t st = w.stream;
    const bool traced = c->trace_log != nullptr;
    long slot = -1;
    if (traced) {
        const long k = c->trace_next.fetch_add(1);
        if (k < c->trace_cap) {
            slot = k;
            std::lock_guard<std::mutex> g(c->trace_mu);
            lpp_trace_step& r = c->trace_steps[k];
            r.worker = worker;
            r.replica = q;
            r.partition = partition;
            r.counter = s_read;
        }
    }
    LAUNCH("args", 0.0, st, lpp::launch_set_step_args(w.args, batch->images, batch->labels, lr, slot, st));
    bool timing;
    {
        std::lock_guard<std::mutex> g(c->timer.mu);
        timing = !c->timer.family.empty();
    }
    if (c->graphs && !timing) {
        // one graph per (worker, partition): snapshot, forward, truncated
        // backward and update, captured once and replayed
        hipGraphExec_t& ge = traced ? w.tgraphs[partition] : w.graphs[partition];
        if (!ge) {
            HIPCHK(hipStreamBeginCapture(st, hipStreamCaptureModeThreadLocal));
            rc = enqueue_step(c, w, worker, partition, traced);
            hipGraph_t graph = nullptr;
            hipError_t e = hipStreamEndCapture(st, &graph);
            if (rc) {
                if (graph) hipGraphDestroy(graph);
                return rc;
            }
            if (e != hipSuccess) return fail(LPP_EHIP, std::string("stream capture: ") + hipGetErrorString(e));
            e = hipGraphInstantiate(&ge, graph, nullptr, nullptr, 0);
            hipGraphDestroy(graph);
            if (e != hipSuccess) {
                ge = nullptr;
                return fail(LPP_EHIP, std::string("graph instantiate: ") + hipGetErrorString(e));
            }
        }
        HIPCHK(hipGraphLaunch(ge, st));
    } else {
        rc = enqueue_step(c, w, worker, partition, traced);
        if (rc) return rc;
    }
    w.last_partition = partition;
    if (c->mode == LPP_SEQUENTIAL) HIPCHK(hipStreamSynchronize(st));
    return LPP_OK;
}

int lpp_average(lpp_ctx* c, const int* replicas, int n_replicas) {
    if (!c) return fail(LPP_EINVAL, "ctx is NULL");
    lpp::RepPtrs rp{};
    int n = 0;
    if (!replicas) {
        if (n_replicas != 0) return fail(LPP_EINVAL, "replicas NULL requires n_replicas == 0");
        for (int q = 0; q < c->K; ++q) rp.p[n++] = c->replicas + (long)q * c->dpad;
    } else {
        if (n_replicas < 1 || n_replicas > c->K) return fail(LPP_EINVAL, "n_replicas out of range");
        std::vector<char> seen(c->K, 0);
        for (int i = 0; i < n_replicas; ++i) {
            const int q = replicas[i];
            if (q < 0 || q >= c->K || seen[q]) return fail(LPP_EINVAL, "replica ids must be distinct and in range");
            seen[q] = 1;
            rp.p[n++] = c->replicas + (long)q * c->dpad;
        }
    }
    if (c->mode == LPP_SEQUENTIAL)
        for (auto& w : c->workers) HIPCHK(hipStreamSynchronize(w.stream));
    hipStream_t st = c->avg_stream;
    long slot = -1;
    if (c->avg_log) {
        const long k = c->avg_next.fetch_add(1);
        if (k < c->trace_cap) {
            slot = k;
            std::lock_guard<std::mutex> g(c->trace_mu);
            lpp_trace_avg& r = c->trace_avgs[k];
            r.index = k;
            r.n_replicas = n;
            r.counter_min = c->counters[0].load();
            for (int q = 1; q < c->K; ++q) r.counter_min = std::min(r.counter_min, c->counters[q].load());
        }
        HIPCHK(lpp::launch_timestamp(c->avg_log, nullptr, slot, 0, st));
    }
    LAUNCH("average", 8.0 * n * c->M.d, st, lpp::launch_average(rp, n, c->M.d, st));
    if (c->avg_log) HIPCHK(lpp::launch_timestamp(c->avg_log, nullptr, slot, 1, st));
    if (c->mode == LPP_SEQUENTIAL) HIPCHK(hipStreamSynchronize(st));
    return LPP_OK;
}

int lpp_sync(lpp_ctx* c) {
    if (!c) return fail(LPP_EINVAL, "ctx is NULL");
    return sync_all(c);
}

int lpp_set_params(lpp_ctx* c, int replica, const float* host, long d) {
    if (!c || !host) return fail(LPP_EINVAL, "NULL argument");
    if (d != c->M.d) return fail(LPP_EINVAL, "d does not match the model");
    if (replica < -1 || replica >= c->K) return fail(LPP_EINVAL, "replica out of range");
    int rc = sync_all(c);
    if (rc) return rc;
    for (int q = 0; q < c->K; ++q)
        if (replica == -1 || replica == q)
            HIPCHK(hipMemcpy(c->replicas + (long)q * c->dpad, host, sizeof(float) * d, hipMemcpyHostToDevice));
    return LPP_OK;
}

int lpp_get_params(lpp_ctx* c, int replica, float* host, long d) {
    if (!c || !host) return fail(LPP_EINVAL, "NULL argument");
    if (d != c->M.d) return fail(LPP_EINVAL, "d does not match the model");
    if (replica < 0 || replica >= c->K) return fail(LPP_EINVAL, "replica out of range");
    int rc = sync_all(c);
    if (rc) return rc;
    HIPCHK(hipMemcpy(host, c->replicas + (long)replica * c->dpad, sizeof(float) * d, hipMemcpyDeviceToHost));
    return LPP_OK;
}

int lpp_get_grad(lpp_ctx* c, int worker, float* host, long d) {
    int rc = check_worker(c, worker);
    if (rc) return rc;
    if (!host || d != c->M.d) return fail(LPP_EINVAL, "bad host buffer or d");
    rc = sync_all(c);
    if (rc) return rc;
    Worker& w = c->workers[worker];
    std::fill(host, host + d, 0.f);
    if (w.last_partition < 0) return LPP_OK;
    const long lo = c->M.blo[w.last_partition], hi = c->M.bhi[w.last_partition];
    HIPCHK(hipMemcpy(host + lo, w.g + lo, sizeof(float) * (hi - lo), hipMemcpyDeviceToHost));
    return LPP_OK;
}

int lpp_get_momentum(lpp_ctx* c, int worker, float* host, long d) {
    int rc = check_worker(c, worker);
    if (rc) return rc;
    if (!host || d != c->M.d) return fail(LPP_EINVAL, "bad host buffer or d");
    rc = sync_all(c);
    if (rc) return rc;
    HIPCHK(hipMemcpy(host, c->workers[worker].m, sizeof(float) * d, hipMemcpyDeviceToHost));
    return LPP_OK;
}

int lpp_set_momentum(lpp_ctx* c, int worker, const float* host, long d) {
    int rc = check_worker(c, worker);
    if (rc) return rc;
    if (!host || d != c->M.d) return fail(LPP_EINVAL, "bad host buffer or d");
    rc = sync_all(c);
    if (rc) return rc;
    HIPCHK(hipMemcpy(c->workers[worker].m, host, sizeof(float) * d, hipMemcpyHostToDevice));
    return LPP_OK;
}

int lpp_get_loss(lpp_ctx* c, int worker, float* loss) {
    int rc = check_worker(c, worker);
    if (rc) return rc;
    if (!loss) return fail(LPP_EINVAL, "loss is NULL");
    rc = sync_all(c);
    if (rc) return rc;
    HIPCHK(hipMemcpy(loss, c->workers[worker].loss, sizeof(float), hipMemcpyDeviceToHost));
    return LPP_OK;
}

int lpp_get_logits(lpp_ctx* c, int worker, float* host, long n) {
    int rc = check_worker(c, worker);
    if (rc) return rc;
    const long want = (long)c->M.desc.batch * c->M.desc.n_classes;
    if (!host || n != want) return fail(LPP_EINVAL, "n must be batch * n_classes");
    rc = sync_all(c);
    if (rc) return rc;
    Worker& w = c->workers[worker];
    HIPCHK(hipMemcpy(host, c->act(w, (int)c->M.layers.size() - 1), sizeof(float) * n, hipMemcpyDeviceToHost));
    return LPP_OK;
}

static int copy_layer_nchw(lpp_ctx* c, int worker, int layer, bool grad, float* host, long n) {
    int rc = check_worker(c, worker);
    if (rc) return rc;
    if (layer < 0 || layer >= (int)c->M.layers.size()) return fail(LPP_EINVAL, "layer out of range");
    const Model& M = c->M;
    const Layer& Y = M.layers[layer];
    const int N = M.desc.batch;
    const long want = (long)N * Y.out.numel();
    if (!host || n != want) return fail(LPP_EINVAL, "n must be batch * c * h * w of the layer");
    Worker& w = c->workers[worker];
    // a fused-away output of a batch-norm group is rebuilt from the group's
    // stored inputs and batch-norm coefficients (the group's own expression
    // without its ReLU; with it for the output of a folded group)
    const Group* G = nullptr;
    bool relu_out = false;   // rebuild with the group's ReLU (a folded group's output)
    if (!grad)
        for (const Group& g : M.groups)
            if (g.kind == G_BNACT && g.fold && layer == g.out) {
                G = &g;
                relu_out = true;
            }
    if (!grad && !M.stored[layer]) {
        for (const Group& g : M.groups)
            if (g.kind == G_BNACT && (layer == g.a || layer == g.add || layer == g.bn2)) G = &g;
        if (!G) return fail(LPP_ESTATE, "this layer's output is fused away (create the context with unfused = 1)");
    }
    if (grad && !M.gstored[layer]) return fail(LPP_ESTATE, "this layer's gradient is fused away");
    if (grad && (w.last_partition < 0 || !M.plans[w.last_partition].run[layer]))
        return fail(LPP_ESTATE, "the last step's backward pass did not reach this layer");
    rc = sync_all(c);
    if (rc) return rc;
    float* tmp = nullptr;
    if (hipMalloc((void**)&tmp, sizeof(float) * n * (G ? 2 : 1)) != hipSuccess)
        return fail(LPP_ENOMEM, "temporary allocation");
    const void* src = grad ? c->dact(w, M.gbuf[layer]) : nullptr;
    hipError_t e = hipSuccess;
    if (G) {
        const int C = Y.out.c;
        const long rows = (long)N * Y.out.h * Y.out.w;
        const int b = layer == G->bn2 ? G->bn2 : G->a;
        const float* ax = c->aux(w, b);
        const void* x = c->act(w, M.layers[b].L.in0);
        const void *r = nullptr, *x2 = nullptr;
        lpp::BnFwd b2{};
        if (layer == G->add) {
            r = G->res >= 0 ? c->act(w, G->res) : nullptr;
            if (G->bn2 >= 0) {
                b2.aux = c->aux(w, G->bn2);
                x2 = c->act(w, M.layers[G->bn2].L.in0);
            }
        }
        lpp::BnFwd b1{};
        b1.aux = (float*)ax;
        e = lpp::launch_bn_act(Y.dt, x, b1, r, x2, x2 ? &b2 : nullptr, relu_out, tmp + n, rows, C, w.stream);
        src = tmp + n;
    } else if (!grad) {
        src = c->act(w, layer);
    }
    if (e == hipSuccess)
        e = lpp::launch_nhwc_to_nchw(Y.dt, src, tmp, N, Y.out.c, Y.out.h, Y.out.w, Y.out.c, w.stream);
    if (e == hipSuccess) e = hipStreamSynchronize(w.stream);
    if (e == hipSuccess) e = hipMemcpy(host, tmp, sizeof(float) * n, hipMemcpyDeviceToHost);
    hipFree(tmp);
    if (e != hipSuccess) return fail(LPP_EHIP, std::string("layer copy: ") + hipGetErrorString(e));
    return LPP_OK;
}

int lpp_get_activation(lpp_ctx* c, int worker, int layer, float* host, long n) {
    return copy_layer_nchw(c, worker, layer, false, host, n);
}

int lpp_get_activation_grad(lpp_ctx* c, int worker, int layer, float* host, long n) {
    return copy_layer_nchw(c, worker, layer, true, host, n);
}

long lpp_num_params(const lpp_ctx* c) { return c ? c->M.d : -1; }

int lpp_block_range(const lpp_ctx* c, int i, long* lo, long* hi) {
    if (!c || !lo || !hi) return fail(LPP_EINVAL, "NULL argument");
    if (i < 0 || i > c->P) return fail(LPP_EINVAL, "block out of range");
    *lo = c->M.blo[i];
    *hi = c->M.bhi[i];
    return LPP_OK;
}

long lpp_counter(const lpp_ctx* c, int replica) {
    if (!c || replica < 0 || replica >= c->K) return -1;
    return c->counters[replica].load();
}

int lpp_timer_enable(lpp_ctx* c, const char* name) {
    if (!c) return fail(LPP_EINVAL, "ctx is NULL");
    int rc = sync_all(c);
    if (rc) return rc;
    std::lock_guard<std::mutex> g(c->timer.mu);
    for (auto& r : c->timer.recs) {
        c->timer.pool.push_back(r.a);
        c->timer.pool.push_back(r.b);
    }
    c->timer.recs.clear();
    c->timer.family = name ? name : "";
    c->timer.ms = c->timer.work = 0;
    c->timer.launches = 0;
    return LPP_OK;
}

int lpp_timer_read(lpp_ctx* c, double* ms, long* launches, double* work) {
    if (!c || !ms || !launches || !work) return fail(LPP_EINVAL, "NULL argument");
    int rc = sync_all(c);
    if (rc) return rc;
    std::lock_guard<std::mutex> g(c->timer.mu);
    for (auto& r : c->timer.recs) {
        float t = 0.f;
        HIPCHK(hipEventElapsedTime(&t, r.a, r.b));
        c->timer.ms += t;
        c->timer.work += r.work;
        c->timer.launches += 1;
        c->timer.pool.push_back(r.a);
        c->timer.pool.push_back(r.b);
    }
    c->timer.recs.clear();
    *ms = c->timer.ms;
    *launches = c->timer.launches;
    *work = c->timer.work;
    return LPP_OK;
}

int lpp_trace_enable(lpp_ctx* c, long capacity) {
    if (!c) return fail(LPP_EINVAL, "ctx is NULL");
    if (capacity < 0 || capacity > (1L << 26)) return fail(LPP_EINVAL, "capacity must be in [0, 2^26]");
    int rc = sync_all(c);
    if (rc) return rc;
    if (c->trace_log) hipFree(c->trace_log);
    if (c->avg_log) hipFree(c->avg_log);
    c->trace_log = c->avg_log = nullptr;
    c->trace_cap = 0;
    c->trace_next.store(0);
    c->avg_next.store(0);
    c->trace_steps.clear();
    c->trace_avgs.clear();
    if (capacity == 0) return LPP_OK;
    const size_t bytes = sizeof(unsigned long long) * 4 * (size_t)capacity;
    if (hipMalloc((void**)&c->trace_log, bytes) != hipSuccess) return fail(LPP_ENOMEM, "trace log allocation");
    if (hipMalloc((void**)&c->avg_log, bytes) != hipSuccess) {
        hipFree(c->trace_log);
        c->trace_log = nullptr;
        return fail(LPP_ENOMEM, "trace log allocation");
    }
    HIPCHK(hipMemset(c->trace_log, 0, bytes));
    HIPCHK(hipMemset(c->avg_log, 0, bytes));
    c->trace_cap = capacity;
    c->trace_steps.assign(capacity, lpp_trace_step{});
    c->trace_avgs.assign(capacity, lpp_trace_avg{});
    return LPP_OK;
}

int lpp_trace_read(lpp_ctx* c, lpp_trace_step* steps, long max_steps, long* n_steps, lpp_trace_avg* avgs,
                   long max_avgs, long* n_avgs) {
    if (!c || !n_steps || !n_avgs) return fail(LPP_EINVAL, "NULL argument");
    if (!c->trace_log) return fail(LPP_ESTATE, "tracing is not enabled");
    int rc = sync_all(c);
    if (rc) return rc;
    const long ns = std::min(c->trace_next.load(), c->trace_cap);
    const long na = std::min(c->avg_next.load(), c->trace_cap);
    *n_steps = ns;
    *n_avgs = na;
    std::vector<unsigned long long> t(4 * (size_t)std::max(ns, na));
    if (steps && ns > 0) {
        if (max_steps < ns) return fail(LPP_EINVAL, "max_steps is smaller than the number of traced steps");
        HIPCHK(hipMemcpy(t.data(), c->trace_log, sizeof(unsigned long long) * 4 * ns, hipMemcpyDeviceToHost));
        std::lock_guard<std::mutex> g(c->trace_mu);
        for (long i = 0; i < ns; ++i) {
            steps[i] = c->trace_steps[i];
            for (int k = 0; k < 4; ++k) steps[i].t[k] = t[4 * i + k];
        }
    }
    if (avgs && na > 0) {
        if (max_avgs < na) return fail(LPP_EINVAL, "max_avgs is smaller than the number of traced rounds");
        HIPCHK(hipMemcpy(t.data(), c->avg_log, sizeof(unsigned long long) * 4 * na, hipMemcpyDeviceToHost));
        std::lock_guard<std::mutex> g(c->trace_mu);
        for (long i = 0; i < na; ++i) {
            avgs[i] = c->trace_avgs[i];
            avgs[i].t[0] = t[4 * i];
            avgs[i].t[1] = t[4 * i + 1];
        }
    }
    return LPP_OK;
}

long lpp_trace_clock_khz(const lpp_ctx* c) {
    if (!c) return -1;
    int khz = 0;
    if (hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, c->device) != hipSuccess) return -1;
    return khz;
}

int lpp_kernel_sgd_update(float* x, float* m, const float* g, long n, float lr, float mu, float wd, void* stream) {
    if (!x || !g || n < 0) return fail(LPP_EINVAL, "bad arguments");
    if (((uintptr_t)x | (uintptr_t)g | (uintptr_t)m) & 15) return fail(LPP_EINVAL, "buffers must be 16-byte aligned");
    hipError_t e = lpp::launch_sgd_update(x, m, g, 0, n, nullptr, lr, mu, wd, (hipStream_t)stream);
    if (e != hipSuccess) return fail(LPP_EHIP, std::string("sgd_update: ") + hipGetErrorString(e));
    return LPP_OK;
}

}  // extern "C"

struct lpp_snap_plan {
    lpp::SnapEntry* tab = nullptr;   // device
    int n_ent = 0;
    long tiles = 0;
    int dt = 0;
    long d = 0;
};

namespace {
// Validates a stand-alone snapshot's conv list (see lpp_snapshot_plan_create)
// into out[0 .. n); returns an error message or nullptr.
const char* snap_convs(const lpp_snap_conv* convs, int n, long d, int dtype, long wbuf_elems,
                       lpp::SnapConvDesc* out) {
    if (dtype != LPP_FP32 && dtype != LPP_BF16) return "unknown dtype";
    if (n < 0 || d < 0 || wbuf_elems < 0 || (n > 0 && !convs)) return "bad arguments";
    const int vw = dtype == LPP_BF16 ? 8 : 4;
    long pos = 0;
    for (int i = 0; i < n; ++i) {
        const lpp_snap_conv& c = convs[i];
        if (c.cout < 1 || c.cin < 1 || c.kh < 1 || c.kw < 1 || c.cin_p < c.cin) return "bad conv shape";
        if (c.cout % vw || c.cin_p % vw) return "cout and cin_p must be multiples of 4 (8 for bf16)";
        const long nw = (long)c.cout * c.cin * c.kh * c.kw;
        if (c.src < pos || c.src + nw > d) return "conv weights must be sorted, disjoint and inside [0, d)";
        pos = c.src + nw;
        const long nf = (long)c.cout * c.kh * c.kw * c.cin_p, nd = (long)c.cin * c.kh * c.kw * c.cout;
        if (c.dst_f < 0 || c.dst_d < 0 || c.dst_f % vw || c.dst_d % vw || c.dst_f + nf > wbuf_elems ||
            c.dst_d + nd > wbuf_elems)
            return "conv layouts must be aligned and inside wbuf";
        out[i] = lpp::SnapConvDesc{c.src, c.cout, c.cin, c.cin_p, c.kh, c.kw, c.dst_f, c.dst_d};
    }
    return nullptr;
}
}  // namespace

extern "C" {

int lpp_snapshot_plan_create(const lpp_snap_conv* convs, int n_convs, long d, int dtype, long wbuf_elems,
                             lpp_snap_plan** out) {
    if (!out) return fail(LPP_EINVAL, "null output pointer");
    *out = nullptr;
    if (n_convs < 0 || n_convs > (1 << 20)) return fail(LPP_EINVAL, "bad conv count");
    std::vector<lpp::SnapConvDesc> cv((size_t)n_convs);
    if (const char* e = snap_convs(convs, n_convs, d, dtype, wbuf_elems, cv.data())) return fail(LPP_EINVAL, e);
    std::vector<lpp::SnapEntry> tab(2 * (size_t)n_convs + 1);
    int n_ent = 0;
    double bytes = 0;
    const long tiles = lpp::snapshot_table(cv.data(), n_convs, d, dtype, tab.data(), (int)tab.size(), &n_ent, &bytes);
    if (tiles < 0) return fail(LPP_EINVAL, "invalid conv list");
    std::unique_ptr<lpp_snap_plan> p(new lpp_snap_plan);
    p->n_ent = n_ent;
    p->tiles = tiles;
    p->dt = dtype;
    p->d = d;
    if (n_ent > 0) {
        if (hipMalloc((void**)&p->tab, sizeof(lpp::SnapEntry) * n_ent) != hipSuccess)
            return fail(LPP_ENOMEM, "snapshot table allocation failed");
        hipError_t e = hipMemcpy(p->tab, tab.data(), sizeof(lpp::SnapEntry) * n_ent, hipMemcpyHostToDevice);
        if (e != hipSuccess) {
            (void)hipFree(p->tab);
            return fail(LPP_EHIP, std::string("snapshot table copy: ") + hipGetErrorString(e));
        }
    }
    *out = p.release();
    return LPP_OK;
}

int lpp_kernel_snapshot(const lpp_snap_plan* plan, const float* x, float* v, void* wbuf, void* stream) {
    if (!plan) return fail(LPP_EINVAL, "null plan");
    if (plan->tiles > 0 && (!x || !v || !wbuf)) return fail(LPP_EINVAL, "null buffer");
    if (((uintptr_t)x | (uintptr_t)v | (uintptr_t)wbuf) & 15) return fail(LPP_EINVAL, "buffers must be 16-byte aligned");
    hipError_t e = lpp::launch_snapshot(plan->dt, x, v, plan->tab, plan->n_ent, plan->tiles, wbuf, (hipStream_t)stream);
    if (e != hipSuccess) return fail(LPP_EHIP, std::string("snapshot: ") + hipGetErrorString(e));
    return LPP_OK;
}

int lpp_kernel_snapshot_noalloc(const lpp_snap_conv* convs, int n_convs, long d, int dtype, long wbuf_elems,
                                const float* x, float* v, void* wbuf, void* stream) {
    if (n_convs < 0 || n_convs > lpp::kSnapNoallocConvs)
        return fail(LPP_EINVAL, "lpp_kernel_snapshot_noalloc takes at most 128 convs");
    lpp::SnapConvDesc cv[lpp::kSnapNoallocConvs];
    if (const char* e = snap_convs(convs, n_convs, d, dtype, wbuf_elems, cv)) return fail(LPP_EINVAL, e);
    if (d > 0 && (!x || !v || !wbuf)) return fail(LPP_EINVAL, "null buffer");
    if (((uintptr_t)x | (uintptr_t)v | (uintptr_t)wbuf) & 15) return fail(LPP_EINVAL, "buffers must be 16-byte aligned");
    int bad = 0;
    hipError_t e = lpp::snapshot_noalloc(dtype, cv, n_convs, d, x, v, wbuf, (hipStream_t)stream, &bad);
    if (bad) return fail(LPP_EINVAL, "invalid conv list");
    if (e != hipSuccess) return fail(LPP_EHIP, std::string("snapshot: ") + hipGetErrorString(e));
    return LPP_OK;
}

int lpp_snapshot_plan_destroy(lpp_snap_plan* plan) {
    if (!plan) return LPP_OK;
    if (plan->tab && hipFree(plan->tab) != hipSuccess) {
        delete plan;
        return fail(LPP_EHIP, "snapshot table free failed");
    }
    delete plan;
    return LPP_OK;
}

int lpp_kernel_average(float* const* replicas, int n_rep, long n, void* stream) {
    if (!replicas || n_rep < 1 || n_rep > lpp::kMaxReplicas || n < 0) return fail(LPP_EINVAL, "bad arguments");
    lpp::RepPtrs rp{};
    for (int k = 0; k < n_rep; ++k) {
        if (!replicas[k] || ((uintptr_t)replicas[k] & 15)) return fail(LPP_EINVAL, "replicas must be 16-byte aligned");
        rp.p[k] = replicas[k];
    }
    hipError_t e = lpp::launch_average(rp, n_rep, n, (hipStream_t)stream);
    if (e != hipSuccess) return fail(LPP_EHIP, std::string("average: ") + hipGetErrorString(e));
    return LPP_OK;
}

}  // extern "C"
