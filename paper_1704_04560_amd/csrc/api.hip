// Host side of the C ABI declared in include/mtx.h: argument validation, the per-model plan
// (layer geometry, flat parameter offsets, workspace carve-up) and the launch sequence of one
// synchronous data-parallel SGD step on the caller's stream.
#include "mtx.h"

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <initializer_list>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "internal.h"

using namespace mtx;

// Workspace of the models created by mtx_init_model_static (see there): one array per device,
// held until the process ends.
constexpr size_t kStaticScratchBytes = (size_t)64 << 20;
static __device__ __align__(256) char scratch[kStaticScratchBytes];

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}

int hip_fail(hipError_t e, const char* what)
{
    return fail(MTX_EHIP, "%s: %s", what, hipGetErrorString(e));
}

#define HIP_TRY(expr, what)                        \
    do {                                           \
        hipError_t _e = (expr);                    \
        if (_e != hipSuccess) return hip_fail(_e, what); \
    } while (0)

constexpr size_t kAlign = 256;
constexpr long long kMaxIndex = 2147483647LL;  // kernels index tensors with 32-bit ints
constexpr long long kMaxBytes = 2147483647LL;  // and read them through 32-bit buffer offsets
constexpr int kFarLimit = 8192;  // spatial sizes stay far below the kernels' out-of-window marker

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

struct LayerPlan {
    int kind, relu;
    int c, h, w, oc, oh, ow, k, s, p, g;
    size_t w_off, w_len, b_off, b_len;
    size_t in_elems, out_elems;  // per sample
    bool act_f32;                // stored output is fp32 (always in fp32 mode; logits)
    bool dgrad_col;              // convolution data gradient through col + col2im
    bool dgrad_fused;            // ... with col tile and col2im in one kernel (dgrad_fused.hip)
    bool need_dx;                // the data gradient of this layer's input is computed
    bool nhwc;                   // stored output is NHWC (convolution and pooling layers)
    int perm_c, perm_hw;         // fully connected after a spatial layer: input in (h, w, c)
    size_t act_off;              // workspace byte offset of the output [B][...]
    size_t dy_off;               // gradient of the loss with respect to that output
    size_t am_off;               // max-pool decisions [B][...] (uint8)
    size_t fw_off, bw_off;       // prepared forward / data-gradient weights (elements)
    bool run;                    // first convolution over the padded input (conv_fwd_run)
    RunGeom rg;                  // its padded input geometry
    int src;                     // residual addition: the layer whose output is added
    bool direct;                 // first convolution through the direct kernels (firstconv.hip)
    size_t stat_off;             // batch normalisation: per-shard (mean, 1/std) [R][C] floats
    size_t skip_off;             // projection shortcut: gradient for the source layer [B][...]
    size_t proj_off;             // projection shortcut: its stored output [B][oh][ow][oc]
    bool dy_shared;              // residual addition: the previous layer's output gradient is
                                 // this layer's own buffer (no copy is made)
};

constexpr size_t kNone = ~(size_t)0;
// blocks of a layer-wise update (it runs beside the backward kernels: a capped grid leaves them
// most of the compute units)
constexpr unsigned kLayerUpdateBlocks = 256;

struct Plan {
    int R = 0, Nb = 0, B = 0, dt = 0;
    int in_c = 0, in_h = 0, in_w = 0;
    size_t P = 0, ld = 0;
    std::vector<LayerPlan> L;
    int first_param = -1;
    bool pool_into_first = false;  // layer 1's max pooling feeds layer 0's direct weight gradient
    bool x_convert = false;      // the input is converted (layout and/or type) before use
    int x_c = 1, x_hw = 1;       // conversion as NCHW -> NHWC with these channels / positions
    std::vector<PrepJob> jobs;   // weight preparation
    int prep_blocks = 0;
    size_t prep_elems = 0;
    size_t xin_off = 0, xin_bytes = 0, prep_off = 0, jobs_off = 0, loss_off = 0;
    size_t partial_off = 0, partial_w_off = 0, col_off = 0, sync_off = 0;
    size_t bn_part_off = 0, bn_coef_off = 0;  // batch normalisation scratch
    size_t first_part_off = 0;                 // direct first convolution: per-image sums
    int n_wgrad = 0;             // layers with a weight gradient
    double gemm_flops = 0;       // multiply-adds x 2 of every matrix launch of a step
    size_t ws_bytes = 0;
};

// The 1x1 convolution of a projection shortcut (layer lp, source sp) over N images.
ConvGeom proj_geom(const LayerPlan& lp, const LayerPlan& sp, int N)
{
    return ConvGeom{N, sp.oc, sp.oh, sp.ow, lp.oc, lp.oh, lp.ow, 1, lp.s, 0, 1};
}

int make_plan(const mtx_model_desc* d, int R, int Nb, Plan& pl)
{
    if (!d) return fail(MTX_EINVAL, "desc is NULL");
    if (!d->layers || d->n_layers < 1) return fail(MTX_EINVAL, "the network has no layers");
    if (d->in_c < 1 || d->in_h < 1 || d->in_w < 1) return fail(MTX_EINVAL, "input shape must be positive");
    if (d->compute != MTX_F32 && d->compute != MTX_BF16) return fail(MTX_EINVAL, "compute must be MTX_F32 or MTX_BF16");
    if (R < 1) return fail(MTX_EINVAL, "R must be >= 1 (got %d)", R);
    if (Nb < 1) return fail(MTX_EINVAL, "shard_batch must be >= 1 (got %d)", Nb);
    const long long B = (long long)R * Nb;
    if (B > kMaxIndex) return fail(MTX_EINVAL, "batch too large");
    pl.R = R; pl.Nb = Nb; pl.B = (int)B; pl.dt = d->compute;
    pl.in_c = d->in_c; pl.in_h = d->in_h; pl.in_w = d->in_w;
    const size_t es = d->compute == MTX_F32 ? 4 : 2;
    if ((long long)d->in_c * d->in_h * d->in_w * B * 4 > kMaxBytes)
        return fail(MTX_EINVAL, "input exceeds 2 GiB");

    int c = d->in_c, h = d->in_h, w = d->in_w;
    size_t off = 0;
    pl.L.clear();
    for (int i = 0; i < d->n_layers; ++i) {
        const mtx_layer& ly = d->layers[i];
        LayerPlan lp{};
        lp.src = -1;
        lp.kind = ly.kind;
        lp.relu = ly.relu ? 1 : 0;
        lp.c = c; lp.h = h; lp.w = w;
        if (ly.kind == MTX_CONV) {
            if (ly.out < 1 || ly.k < 1 || ly.stride < 1 || ly.pad < 0 || ly.groups < 1)
                return fail(MTX_EINVAL, "layer %d: invalid convolution parameters", i);
            if (c % ly.groups || ly.out % ly.groups)
                return fail(MTX_EINVAL, "layer %d: groups must divide both channel counts", i);
            if (h + 2 * ly.pad < ly.k || w + 2 * ly.pad < ly.k)
                return fail(MTX_EINVAL, "layer %d: kernel larger than the padded input", i);
            lp.k = ly.k; lp.s = ly.stride; lp.p = ly.pad; lp.g = ly.groups;
            lp.oc = ly.out;
            lp.oh = (h + 2 * ly.pad - ly.k) / ly.stride + 1;
            lp.ow = (w + 2 * ly.pad - ly.k) / ly.stride + 1;
            lp.w_len = (size_t)ly.out * (c / ly.groups) * ly.k * ly.k;
            lp.b_len = ly.out;
        } else if (ly.kind == MTX_FC) {
            if (ly.out < 1) return fail(MTX_EINVAL, "layer %d: out must be >= 1", i);
            if ((ly.k != 0 && ly.k != 1) || (ly.stride != 0 && ly.stride != 1) || ly.pad != 0 ||
                (ly.groups != 0 && ly.groups != 1))
                return fail(MTX_EINVAL, "layer %d: a fully connected layer takes only out and relu", i);
            lp.k = 1; lp.s = 1; lp.p = 0; lp.g = 1;
            lp.oc = ly.out; lp.oh = 1; lp.ow = 1;
            lp.w_len = (size_t)ly.out * c * h * w;
            lp.b_len = ly.out;
        } else if (ly.kind == MTX_MAXPOOL) {
            if (ly.k < 1 || ly.k > 16 || ly.stride < 1)
                return fail(MTX_EINVAL, "layer %d: pooling needs 1 <= k <= 16 and stride >= 1", i);
            if (ly.out != 0 || ly.pad != 0 || ly.relu || (ly.groups != 0 && ly.groups != 1))
                return fail(MTX_EINVAL, "layer %d: pooling takes only k and stride", i);
            if (h < ly.k || w < ly.k) return fail(MTX_EINVAL, "layer %d: window larger than the input", i);
            lp.k = ly.k; lp.s = ly.stride; lp.p = 0; lp.g = 1;
            lp.oc = c;
            lp.oh = (h - ly.k) / ly.stride + 1;
            lp.ow = (w - ly.k) / ly.stride + 1;
            lp.w_len = 0; lp.b_len = 0;
        } else if (ly.kind == MTX_BN) {
            if ((ly.out != 0 && ly.out != c) || ly.k != 0 || ly.pad != 0 ||
                (ly.stride != 0 && ly.stride != 1) || (ly.groups != 0 && ly.groups != 1))
                return fail(MTX_EINVAL, "layer %d: batch normalisation takes only relu (out, if "
                                        "given, must be its channel count)", i);
            const int vw = 16 / (int)es;
            if (c > 256 && !(c % vw == 0 && c / vw <= 256))
                return fail(MTX_EUNSUPPORTED, "layer %d: batch normalisation of %d channels (more "
                                              "than 256 need a multiple of %d, at most %d)",
                            i, c, vw, 256 * vw);
            lp.k = 1; lp.s = 1; lp.p = 0; lp.g = 1;
            lp.oc = c; lp.oh = h; lp.ow = w;
            lp.w_len = c; lp.b_len = c;  // gamma, beta
        } else if (ly.kind == MTX_ADD || ly.kind == MTX_ADDP) {
            const int src = ly.k;
            if (src < 0 || src > i - 2)
                return fail(MTX_EINVAL, "layer %d: the added layer must be an earlier layer "
                                        "other than the previous one", i);
            const LayerPlan& sp = pl.L[src];
            for (int j = src + 1; j < i; ++j)
                if ((pl.L[j].kind == MTX_ADD || pl.L[j].kind == MTX_ADDP) && pl.L[j].src == src)
                    return fail(MTX_EINVAL, "layer %d: layer %d is already added once", i, src);
            if (ly.kind == MTX_ADD) {
                if (sp.oc != c || sp.oh != h || sp.ow != w)
                    return fail(MTX_EINVAL, "layer %d: layer %d's output has another shape", i, src);
                if (ly.out != 0 || ly.pad != 0 || (ly.stride != 0 && ly.stride != 1) ||
                    (ly.groups != 0 && ly.groups != 1))
                    return fail(MTX_EINVAL, "layer %d: a residual addition takes only k and relu", i);
                lp.s = 1;
                lp.w_len = 0; lp.b_len = 0;
            } else {
                const int st = ly.stride;
                if (st < 1 || ly.out != c || ly.pad != 0 || (ly.groups != 0 && ly.groups != 1))
                    return fail(MTX_EINVAL, "layer %d: a projection shortcut takes k, out (the "
                                            "previous layer's channel count), stride >= 1 and relu", i);
                if ((sp.oh - 1) / st + 1 != h || (sp.ow - 1) / st + 1 != w)
                    return fail(MTX_EINVAL, "layer %d: a 1x1 convolution of stride %d does not map "
                                            "layer %d's output to this layer's shape", i, st, src);
                lp.s = st;
                lp.w_len = (size_t)c * sp.oc;  // W[out][c of the source], 1x1
                lp.b_len = c;
            }
            lp.src = src;
            lp.k = 1; lp.p = 0; lp.g = 1;
            lp.oc = c; lp.oh = h; lp.ow = w;
        } else {
            return fail(MTX_EINVAL, "layer %d: unknown kind %d", i, ly.kind);
        }
        lp.in_elems = (size_t)c * h * w;
        lp.out_elems = (size_t)lp.oc * lp.oh * lp.ow;
        if ((long long)lp.out_elems * B * 4 > kMaxBytes || (long long)lp.w_len * 4 > kMaxBytes)
            return fail(MTX_EINVAL, "layer %d: a tensor exceeds 2 GiB", i);
        lp.w_off = off; off += lp.w_len;
        lp.b_off = off; off += lp.b_len;
        if (lp.w_len && pl.first_param < 0) pl.first_param = i;
        pl.L.push_back(lp);
        c = lp.oc; h = lp.oh; w = lp.ow;
    }
    const LayerPlan& last = pl.L.back();
    if (last.kind != MTX_FC || last.relu)
        return fail(MTX_EINVAL, "the last layer must be fully connected without ReLU (class scores)");
    pl.P = off;
    pl.ld = align_up(off, 64);

    // which layers propagate a data gradient, output layouts, input permutations
    for (size_t i = 0; i < pl.L.size(); ++i) {
        LayerPlan& lp = pl.L[i];
        lp.need_dx = (int)i > pl.first_param && pl.first_param >= 0;
        // a pooled tensor that feeds a fully connected layer is stored NCHW
        lp.nhwc = lp.kind == MTX_CONV || lp.kind == MTX_BN || lp.kind == MTX_ADD ||
                  lp.kind == MTX_ADDP ||
                  (lp.kind == MTX_MAXPOOL && !(i + 1 < pl.L.size() && pl.L[i + 1].kind == MTX_FC));
        lp.perm_c = 1;
        lp.perm_hw = 1;
        if (lp.kind == MTX_FC && i > 0 && pl.L[i - 1].nhwc && lp.c > 1 && lp.h * lp.w > 1) {
            lp.perm_c = lp.c;
            lp.perm_hw = lp.h * lp.w;
        }
        if (lp.kind != MTX_FC && (lp.h >= kFarLimit || lp.w >= kFarLimit))
            return fail(MTX_EINVAL, "layer %d: spatial size must be below %d", (int)i, kFarLimit);
    }
    LayerPlan& first = pl.L.front();
    if (first.kind == MTX_FC) {
        pl.x_c = 1;
        pl.x_hw = (int)first.in_elems;
    } else {
        pl.x_c = pl.in_c;
        pl.x_hw = pl.in_h * pl.in_w;
    }
    pl.x_convert = pl.dt == MTX_BF16 || (pl.x_c > 1 && pl.x_hw > 1);
    // A first convolution whose channel count rules out 16-byte loads reads a padded input
    // instead (see conv_fwd_run), when that adds at most 3x to its multiply-adds.
    first.run = false;
    if (first.kind == MTX_CONV && first.g == 1 && first.c % vec_elems(pl.dt) != 0) {
        const int vecb = 16 / (int)es;  // elements per 16 bytes
        int cp = first.c;
        while ((first.s * cp) % vecb) ++cp;
        const int run = (first.k * cp + vecb - 1) / vecb * vecb;
        int wp = first.w + 2 * first.p;
        while ((wp * cp) % vecb) ++wp;
        const double inflate = (double)first.k * run / ((double)first.k * first.k * first.c);
        if (inflate <= 3.0) {
            first.run = true;
            first.rg = RunGeom{first.h + 2 * first.p, wp, cp, run};
            pl.x_convert = true;
        }
    }
    // A first convolution of one input channel with a small window runs as direct kernels.
    first.direct = false;
    if (first.kind == MTX_CONV && !first.run) {
        const ConvGeom g0{pl.B, first.c, first.h, first.w, first.oc, first.oh, first.ow, first.k,
                          first.s, first.p, first.g};
        first.direct = first_conv_direct(g0, pl.dt);
    }
    // A max pooling right above such a layer (window = stride, NHWC output) hands its output
    // gradient and decisions to the direct weight-gradient kernel, which forms the layer's output
    // gradient itself: the pooling backward launch goes away.
    pl.pool_into_first = false;
    if (first.direct && pl.L.size() > 2) {
        const LayerPlan& p1 = pl.L[1];
        bool kept_for_0 = false;  // a residual addition whose source is layer 0
        for (const LayerPlan& q : pl.L)
            kept_for_0 = kept_for_0 || ((q.kind == MTX_ADD || q.kind == MTX_ADDP) && q.src == 0);
        const ConvGeom g0{pl.B, first.c, first.h, first.w, first.oc, first.oh, first.ow, first.k,
                          first.s, first.p, first.g};
        pl.pool_into_first = p1.kind == MTX_MAXPOOL && p1.k == p1.s && p1.nhwc && !kept_for_0 &&
                             first_conv_pool_ok(g0, p1.k);
    }

    // weight preparation jobs; every prepared tensor starts 16-byte aligned
    size_t pe = 0;
    int blocks = 0;
    pl.jobs.clear();
    auto add_job = [&](PrepJob j) {
        j.dst = (long long)pe;
        j.block0 = blocks;
        prep_fill_divisors(j);
        blocks += prep_blocks(j.n);
        pe = align_up(pe + (size_t)j.n, 8);
        pl.jobs.push_back(j);
        return (size_t)j.dst;
    };
    for (size_t i = 0; i < pl.L.size(); ++i) {
        LayerPlan& lp = pl.L[i];
        lp.fw_off = lp.bw_off = kNone;
        if (!lp.w_len || lp.kind == MTX_BN) continue;  // BN reads gamma and beta as they are
        PrepJob j{};
        j.n = (int)lp.w_len;
        j.src = (long long)lp.w_off;
        if (lp.kind == MTX_CONV && lp.run) {
            j.kind = PREP_CONV_RUN;
            j.n = lp.oc * lp.k * lp.rg.RUN;
            j.C = lp.c; j.Cp = lp.rg.Cp; j.K = lp.k; j.RUN = lp.rg.RUN;
            lp.fw_off = add_job(j);
        } else if (lp.kind == MTX_CONV && lp.direct) {
            continue;  // the direct kernels read the fp32 weights (and round them as they load)
        } else if (lp.kind == MTX_ADDP) {
            // the projection's 1x1 convolution: forward layout, and the data-gradient layout
            // when the source's gradient is needed (its data gradient is an implicit GEMM)
            j.g = 1; j.cg = pl.L[lp.src].oc; j.og = lp.oc; j.KK = 1;
            j.kind = PREP_CONV_F;
            lp.fw_off = add_job(j);
            if (lp.src >= pl.first_param) {
                lp.dgrad_col = conv_dgrad_use_col(proj_geom(lp, pl.L[lp.src], pl.B));
                j.kind = lp.dgrad_col ? PREP_CONV_C : PREP_CONV_D;
                lp.bw_off = add_job(j);
            }
        } else if (lp.kind == MTX_CONV) {
            j.g = lp.g; j.cg = lp.c / lp.g; j.og = lp.oc / lp.g; j.KK = lp.k * lp.k;
            j.kind = PREP_CONV_F;
            lp.fw_off = add_job(j);
            if (lp.need_dx) {
                ConvGeom gb{pl.B, lp.c, lp.h, lp.w, lp.oc, lp.oh, lp.ow, lp.k, lp.s, lp.p, lp.g};
                lp.dgrad_col = conv_dgrad_use_col(gb);
                lp.dgrad_fused = lp.dgrad_col && conv_dgrad_fused_ok(gb, pl.dt);
                j.kind = lp.dgrad_col ? PREP_CONV_C : PREP_CONV_D;
                if (!lp.dgrad_fused) lp.bw_off = add_job(j);  // the fused kernel reads W itself
            }
        } else {
            if (lp.perm_c > 1) {
                j.kind = PREP_FC_PERM;
                j.C = lp.perm_c; j.HW = lp.perm_hw; j.IN = (int)lp.in_elems;
            } else {
                j.kind = PREP_CAST;
            }
            lp.fw_off = add_job(j);
            lp.bw_off = lp.fw_off;
        }
    }
    pl.prep_blocks = blocks;
    pl.prep_elems = pe;

    // workspace carve-up
    size_t ws = 0;
    // fp32 partial sums: one region for the forward and data-gradient launches, one for the
    // weight gradients (which may run concurrently on a second stream)
    size_t max_partial = 0, max_partial_w = 0, max_col = 0, max_bn_part = 0, max_bn_coef = 0;
    size_t max_first = 0;
    for (size_t i = 0; i < pl.L.size(); ++i) {
        LayerPlan& lp = pl.L[i];
        lp.act_f32 = (pl.dt == MTX_F32) || (i + 1 == pl.L.size());
        lp.act_off = ws;
        ws = align_up(ws + lp.out_elems * pl.B * (lp.act_f32 ? 4 : es), kAlign);
        if (lp.kind == MTX_MAXPOOL) {
            lp.am_off = ws;
            ws = align_up(ws + lp.out_elems * pl.B, kAlign);
        }
        if ((int)i >= pl.first_param) {
            lp.dy_off = ws;
            ws = align_up(ws + lp.out_elems * pl.B * es, kAlign);
        }
        if (lp.kind == MTX_BN) {
            lp.stat_off = ws;
            ws = align_up(ws + (size_t)pl.R * lp.c * kBnStatFloats * 4, kAlign);
            max_bn_part = std::max(max_bn_part, bn_partial_doubles((Dt)pl.dt, pl.R, lp.c, pl.Nb,
                                                                   lp.h * lp.w));
            max_bn_coef = std::max(max_bn_coef, (size_t)pl.R * lp.c * 3);
        }
        // a projection shortcut keeps the gradient for its source (its data gradient) until the
        // source's own output gradient exists (only when the source's gradient is needed at
        // all); an identity addition's share is its own output gradient, which stays unchanged
        // until the end of the step, so it needs no buffer of its own
        lp.skip_off = kNone;
        if (lp.kind == MTX_ADDP && lp.src >= pl.first_param && pl.first_param >= 0) {
            lp.skip_off = ws;
            ws = align_up(ws + pl.L[lp.src].out_elems * pl.B * es, kAlign);
        }
        lp.proj_off = kNone;
        if (lp.kind == MTX_ADDP) {
            lp.proj_off = ws;
            ws = align_up(ws + lp.out_elems * pl.B * (lp.act_f32 ? 4 : es), kAlign);
        }
        // fp32 partial sums of the matrix launches whose reduction is split (the last entry of
        // dims is the weight gradient)
        GemmDims dims[3];
        int nd = 0;
        if (lp.kind == MTX_CONV && lp.direct) {
            ConvGeom gs{pl.Nb, lp.c, lp.h, lp.w, lp.oc, lp.oh, lp.ow, lp.k, lp.s, lp.p, lp.g};
            max_first = std::max(max_first, first_conv_partial_floats(gs, pl.R));
        } else if (lp.kind == MTX_CONV) {
            ConvGeom gb{pl.B, lp.c, lp.h, lp.w, lp.oc, lp.oh, lp.ow, lp.k, lp.s, lp.p, lp.g};
            ConvGeom gs = gb;
            gs.N = pl.Nb;
            dims[nd++] = lp.run ? conv_fwd_run_dims(pl.dt, gb, lp.rg) : conv_fwd_dims(pl.dt, gb);
            if (lp.need_dx) {
                if (lp.dgrad_fused) {
                    // no col buffer and no split reduction
                } else if (lp.dgrad_col) {
                    dims[nd++] = conv_dgrad_col_dims(pl.dt, gb);
                    if (conv_dgrad_col_elems(gb) > max_col) max_col = conv_dgrad_col_elems(gb);
                } else {
                    dims[nd++] = conv_dgrad_dims(pl.dt, gb);
                }
            }
            dims[nd++] = lp.run ? conv_wgrad_run_dims(pl.dt, gs, lp.rg, pl.R)
                                : conv_wgrad_dims(pl.dt, gs, pl.R);
        } else if (lp.kind == MTX_FC) {
            dims[nd++] = fc_fwd_dims(pl.dt, pl.B, (int)lp.in_elems, lp.oc);
            if (lp.need_dx) dims[nd++] = fc_dgrad_dims(pl.dt, pl.B, (int)lp.in_elems, lp.oc);
            dims[nd++] = fc_wgrad_dims(pl.dt, pl.Nb, pl.R, (int)lp.in_elems, lp.oc);
        } else if (lp.kind == MTX_ADDP) {
            const LayerPlan& sp = pl.L[lp.src];
            const ConvGeom gp = proj_geom(lp, sp, pl.B);
            dims[nd++] = conv_fwd_dims(pl.dt, gp);
            if (lp.src >= pl.first_param && lp.dgrad_col) {
                dims[nd++] = conv_dgrad_col_dims(pl.dt, gp);
                if (conv_dgrad_col_elems(gp) > max_col) max_col = conv_dgrad_col_elems(gp);
            } else if (lp.src >= pl.first_param) {
                dims[nd++] = conv_dgrad_dims(pl.dt, gp);
            }
            dims[nd++] = conv_wgrad_dims(pl.dt, proj_geom(lp, sp, pl.Nb), pl.R);
        }
        for (int k = 0; k < nd; ++k) {
            const size_t pz = partial_elems(pl.dt, dims[k]);
            const bool wgrad = k == nd - 1;
            size_t& mx = wgrad ? max_partial_w : max_partial;
            if (pz > mx) mx = pz;
            // the first parameter layer's weight gradient runs on the caller's stream
            if (wgrad && (int)i == pl.first_param && pz > max_partial) max_partial = pz;
        }
        if (lp.w_len) pl.n_wgrad += 1;
        if (lp.w_len && lp.kind == MTX_ADDP) {
            const double macs = (double)pl.B * lp.oh * lp.ow * lp.oc * pl.L[lp.src].oc;
            pl.gemm_flops += 2.0 * macs * (lp.src >= pl.first_param ? 3 : 2);
        } else if (lp.w_len && lp.kind != MTX_BN) {
            const double macs = lp.kind == MTX_CONV
                                    ? (double)pl.B * lp.oh * lp.ow * lp.oc * (lp.c / lp.g) * lp.k * lp.k
                                    : (double)pl.B * lp.in_elems * lp.oc;
            pl.gemm_flops += 2.0 * macs * (lp.need_dx ? 3 : 2);
        }
    }
    // A residual addition passes its output gradient to the previous layer unchanged when that
    // layer has no ReLU (its output is not read by any other addition): the previous layer then
    // reads the addition's gradient buffer itself instead of a copy (the batch normalisation
    // before each addition of the residual networks: one tensor written and read less).
    for (size_t i = 1; i < pl.L.size(); ++i) {
        LayerPlan& lp = pl.L[i];
        lp.dy_shared = false;
        if ((lp.kind != MTX_ADD && lp.kind != MTX_ADDP) || !lp.need_dx || pl.L[i - 1].relu)
            continue;
        bool other = false;
        for (size_t j = 0; j < pl.L.size(); ++j)
            if ((pl.L[j].kind == MTX_ADD || pl.L[j].kind == MTX_ADDP) &&
                pl.L[j].src == (int)i - 1)
                other = true;
        if (other) continue;
        pl.L[i - 1].dy_off = lp.dy_off;
        lp.dy_shared = true;
    }
    if (pl.x_convert) {
        pl.xin_off = ws;
        const size_t xe = first.run ? (size_t)first.rg.Hp * first.rg.Wp * first.rg.Cp
                                    : (size_t)pl.in_c * pl.in_h * pl.in_w;
        if ((long long)xe * pl.B * es > kMaxBytes) return fail(MTX_EINVAL, "input exceeds 2 GiB");
        pl.xin_bytes = xe * pl.B * es;
        ws = align_up(ws + pl.xin_bytes, kAlign);
    }
    pl.prep_off = ws;
    ws = align_up(ws + pl.prep_elems * es, kAlign);
    pl.jobs_off = ws;
    ws = align_up(ws + pl.jobs.size() * sizeof(PrepJob), kAlign);
    pl.loss_off = ws;  // per-block loss sums of the softmax launch, then its counter
    pl.sync_off = align_up(ws + (size_t)((pl.B + 3) / 4) * 4, kAlign);
    ws = pl.sync_off + kAlign;
    pl.partial_off = ws;
    ws = align_up(ws + max_partial * 4, kAlign);
    pl.partial_w_off = ws;
    ws = align_up(ws + max_partial_w * 4, kAlign);
    pl.col_off = ws;
    ws = align_up(ws + max_col * 4, kAlign);
    pl.bn_part_off = ws;
    ws = align_up(ws + max_bn_part * 8, kAlign);
    pl.first_part_off = ws;
    ws = align_up(ws + max_first * 4, kAlign);
    pl.bn_coef_off = ws;
    ws = align_up(ws + max_bn_coef * 4, kAlign);
    pl.ws_bytes = ws;
    return MTX_OK;
}

// ---- the static workspace of mtx_init_model_static ------------------------------------------
// A model created by mtx_init_model_static runs its steps in this array instead of a caller
// workspace.  Host code must never pass the array's name to a kernel or a copy (on the host it
// is only a stand-in symbol): the device address comes from hipGetSymbolAddress, once per
// device, and is kept in g_scratch_ptr.
constexpr int kStaticMaxJobs = 16;  // weight-preparation jobs re-written by every static step
constexpr int kMaxDevices = 64;

std::mutex g_scratch_mu;
char* g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on the current device (resolved on first use).
int static_scratch(char** out)
{
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices) return fail(MTX_EUNSUPPORTED, "device %d out of range", dev);
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* ptr = nullptr;
        e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !ptr) return hip_fail(e, "hipGetSymbolAddress(scratch)");
        g_scratch_ptr[dev] = static_cast<char*>(ptr);
    }
    *out = g_scratch_ptr[dev];
    return MTX_OK;
}

// What a static model re-establishes in the shared array before each step: its weight
// preparation jobs, the zero loss counter, and (a first convolution over a padded input) the
// zero padded input whose border the step never writes.
struct StaticSetup {
    PrepJob jobs[kStaticMaxJobs];
    int njobs;
    PrepJob* dst_jobs;
    unsigned* sync;
    uint4* zero;
    unsigned long long zero_vecs;  // 16-byte vectors to clear at `zero`
};

__global__ __launch_bounds__(256) void static_setup_kernel(const StaticSetup a)
{
    const unsigned long long tid = (unsigned long long)blockIdx.x * blockDim.x + threadIdx.x;
    const unsigned long long nth = (unsigned long long)gridDim.x * blockDim.x;
    if (blockIdx.x == 0) {
        for (int j = threadIdx.x; j < a.njobs; j += blockDim.x) a.dst_jobs[j] = a.jobs[j];
        if (threadIdx.x == 0) *a.sync = 0u;
    }
    for (unsigned long long i = tid; i < a.zero_vecs; i += nth) a.zero[i] = uint4{0u, 0u, 0u, 0u};
}

// First output of a SplitMix64 generator whose state is `key` (Steele, Lea & Flood 2014;
// constants of Vigna's splitmix64.c).
uint64_t splitmix64_first(uint64_t key)
{
    uint64_t z = key + 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

void glorot_init_host(const Plan& pl, uint64_t seed, std::vector<float>& w)
{
    w.assign(pl.P, 0.0f);
    for (size_t l = 0; l < pl.L.size(); ++l) {
        const LayerPlan& lp = pl.L[l];
        if (!lp.w_len) continue;
        if (lp.kind == MTX_BN) {  // gamma = 1, beta = 0: the identity at the start
            for (size_t i = 0; i < lp.w_len; ++i) w[lp.w_off + i] = 1.0f;
            continue;
        }
        double fan_in, fan_out;
        if (lp.kind == MTX_CONV) {
            fan_in = (double)(lp.c / lp.g) * lp.k * lp.k;
            fan_out = (double)lp.oc * lp.k * lp.k;
        } else if (lp.kind == MTX_ADDP) {  // a 1x1 convolution of the source's channels
            fan_in = (double)pl.L[lp.src].oc;
            fan_out = (double)lp.oc;
        } else {
            fan_in = (double)lp.in_elems;
            fan_out = (double)lp.oc;
        }
        const double a = std::sqrt(6.0 / (fan_in + fan_out));
        for (size_t i = 0; i < lp.w_len; ++i) {
            const uint64_t hsh = splitmix64_first(seed ^ (((uint64_t)l << 32) | (uint64_t)i));
            const double u = (double)(hsh >> 40) / 16777216.0;
            w[lp.w_off + i] = (float)(a * (2.0 * u - 1.0));
        }
    }
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

bool overlap(const void* a, size_t abytes, const void* b, size_t bbytes)
{
    const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
    return x < y + bbytes && y < x + abytes;
}

}  // namespace

// Optional per-launch timing: every launch site of the step owns a small ring of event pairs;
// a pair is read back (and its time accumulated) before it is reused or when asked for.
struct Timer {
    static constexpr int kDepth = 4;
    struct Site {
        std::string name;
        int layer = -1;
        hipEvent_t ev[kDepth][2] = {};
        int head = 0, pending = 0;
        long launches = 0;
        double ms = 0.0;
    };
    bool on = false;
    int cur = 0;
    std::vector<Site> sites;

    hipError_t retire(Site& st)
    {
        const int slot = (st.head - st.pending + kDepth) % kDepth;
        hipError_t e = hipEventSynchronize(st.ev[slot][1]);
        float ms = 0.f;
        if (e == hipSuccess) e = hipEventElapsedTime(&ms, st.ev[slot][0], st.ev[slot][1]);
        if (e != hipSuccess) return e;
        st.ms += ms;
        st.launches += 1;
        st.pending -= 1;
        return hipSuccess;
    }
    hipError_t drain()
    {
        for (auto& st : sites)
            while (st.pending) {
                hipError_t e = retire(st);
                if (e != hipSuccess) return e;
            }
        return hipSuccess;
    }
    void destroy()
    {
        for (auto& st : sites)
            for (auto& pr : st.ev)
                for (auto& e : pr)
                    if (e) (void)hipEventDestroy(e);
        sites.clear();
    }
};

// Replay of a captured step.  The launch sequence of mtx_train_step depends only on the model
// and on (x, labels, lr, momentum, loss_out); it is captured once into a HIP graph on a private
// stream and replayed on the caller's stream while those arguments stay the same.
struct GraphCache {
    bool enabled = false;
    hipStream_t capture_stream = nullptr;
    hipGraphExec_t exec = nullptr;
    const float* x = nullptr;
    const int32_t* labels = nullptr;
    float lr = 0.f, mu = 0.f;
    float* loss = nullptr;
    int misses = 0;  // consecutive captures; replay is abandoned after kMaxMisses
    static constexpr int kMaxMisses = 3;
    bool matches(const float* x_, const int32_t* l_, float lr_, float mu_, float* loss_) const
    {
        return exec && x == x_ && labels == l_ && lr == lr_ && mu == mu_ && loss == loss_;
    }
    void reset()
    {
        if (exec) (void)hipGraphExecDestroy(exec);
        exec = nullptr;
    }
    void destroy()
    {
        reset();
        if (capture_stream) (void)hipStreamDestroy(capture_stream);
        capture_stream = nullptr;
    }
};

struct mtx_model {
    Plan pl;
    float* w;
    float* v;
    float* grads;
    float* gavg;
    char* ws;
    hipStream_t last_stream;
    Timer timer;
    GraphCache graph;
    // second stream for the weight gradients (overlapped with the data-gradient chain), third
    // stream for the layer-wise average + update that follows each layer's weight gradients
    bool overlap = false;
    hipStream_t side = nullptr;
    std::vector<hipEvent_t> fork;  // per weight-gradient launch: its output gradient is ready
    hipEvent_t join = nullptr;     // every weight gradient is done
    bool layerwise = false;         // average + update per layer on the third stream
    hipStream_t upd = nullptr;
    std::vector<hipEvent_t> wdone;  // per parameter layer: its weight gradients are done
    std::vector<hipEvent_t> ddone;  // per parameter layer: the kernels on the caller's stream
                                    // that read its master weights are done
    hipEvent_t upd_join = nullptr;  // every layer's update is done
    // the fully connected layers at the end of the parameter list carry their own average +
    // update in their weight-gradient launch (mtx_set_fused_update)
    bool fuse_update = true;
    // the non-finite check (mtx_set_nonfinite_check): average, flag, update unless flagged
    bool check_finite = false;
    // update rule after the average (mtx_set_optimizer): momentum, or Adam / AdaGrad with their
    // first state in v, Adam's second moment in s2, and the number of steps taken since
    int opt = MTX_OPT_MOMENTUM;
    float b1 = 0.9f, b2 = 0.999f, eps = 0.0f;
    float* s2 = nullptr;
    long long opt_step = 0;
    // matrix launches of the last enqueued step (mtx_get_launches)
    std::vector<mtx_launch_info> launches;
    // the workspace is the device's static array (mtx_init_model_static), shared with every
    // other static model on the device: each step re-establishes what it needs there first
    bool static_ws = false;
};

namespace {

// Timing context of the launch site being enqueued (timing runs are single-threaded per model;
// the context lives only while a site's launches are enqueued).
struct TimingCtx {
    mtx_model* m = nullptr;
    std::string base;
    int layer = -1;
    int site = -1;
};
thread_local TimingCtx g_tctx;

// Start site number t.cur (creating it on the first step), recording its start event.
hipError_t begin_site(mtx_model* m, const std::string& name, int layer, hipStream_t s, int* idx)
{
    Timer& t = m->timer;
    if ((int)t.sites.size() <= t.cur) {
        Timer::Site st;
        st.name = name;
        st.layer = layer;
        for (auto& pr : st.ev)
            for (auto& e : pr) {
                hipError_t err = hipEventCreate(&e);
                if (err != hipSuccess) return err;
            }
        t.sites.push_back(st);
    }
    *idx = t.cur++;
    Timer::Site& st = t.sites[*idx];
    if (st.pending == Timer::kDepth) {
        hipError_t e = t.retire(st);
        if (e != hipSuccess) return e;
    }
    return hipEventRecord(st.ev[st.head][0], s);
}

hipError_t end_site(mtx_model* m, int idx, hipStream_t s)
{
    Timer::Site& st = m->timer.sites[idx];
    hipError_t e = hipEventRecord(st.ev[st.head][1], s);
    if (e != hipSuccess) return e;
    st.head = (st.head + 1) % Timer::kDepth;
    st.pending += 1;
    return hipSuccess;
}

// Run one launch site (a callable returning hipError_t); with timing on, bracket it with an
// event pair.  A site that launches several kernels marks the boundaries with timing_split, so
// that every kernel is timed on its own.
// Site whose launches are being enqueued, for the launch record.
struct RecordCtx {
    mtx_model* m = nullptr;
    const char* name = nullptr;
    int layer = -1;
};
thread_local RecordCtx g_rec;

template <class F>
hipError_t launch_site(mtx_model* m, const char* name, int layer, hipStream_t s, F&& f)
{
    g_rec = RecordCtx{m, name, layer};
    struct Clear {
        ~Clear() { g_rec = RecordCtx{}; }
    } clear;
    if (!m->timer.on) return f();
    g_tctx.m = m;
    g_tctx.base = name;
    g_tctx.layer = layer;
    hipError_t e = begin_site(m, name, layer, s, &g_tctx.site);
    if (e == hipSuccess) e = f();
    if (e == hipSuccess) e = end_site(m, g_tctx.site, s);
    g_tctx.m = nullptr;
    return e;
}

}  // namespace

namespace {
void release_update_stream(mtx_model* m)
{
    for (hipEvent_t& e : m->wdone)
        if (e) (void)hipEventDestroy(e);
    m->wdone.clear();
    for (hipEvent_t& e : m->ddone)
        if (e) (void)hipEventDestroy(e);
    m->ddone.clear();
    if (m->upd_join) (void)hipEventDestroy(m->upd_join);
    m->upd_join = nullptr;
    if (m->upd) (void)hipStreamDestroy(m->upd);
    m->upd = nullptr;
}

void destroy_streams(mtx_model* m)
{
    for (hipEvent_t& e : m->fork)
        if (e) (void)hipEventDestroy(e);
    m->fork.clear();
    if (m->join) (void)hipEventDestroy(m->join);
    m->join = nullptr;
    if (m->side) (void)hipStreamDestroy(m->side);
    m->side = nullptr;
    release_update_stream(m);
}
}  // namespace

namespace mtx {
void note_gemm(int fp, int fq, int bk, int splits, int flags)
{
    const RecordCtx& r = g_rec;
    if (!r.m) return;
    mtx_launch_info li{};
    std::snprintf(li.site, sizeof li.site, "%s", r.name);
    li.layer = r.layer;
    li.tile_rows = 32 * fp;
    li.tile_cols = 32 * fq;
    li.k_tile = bk;
    li.splits = splits;
    li.flags = flags;
    r.m->launches.push_back(li);
}

void timing_split(hipStream_t s, const char* part)
{
    TimingCtx& c = g_tctx;
    if (!c.m) return;
    if (end_site(c.m, c.site, s) != hipSuccess) return;
    if (begin_site(c.m, c.base + "_" + part, c.layer, s, &c.site) != hipSuccess) c.m = nullptr;
}
}  // namespace mtx

extern "C" {

const char* mtx_last_error(void) { return g_err.c_str(); }

int mtx_model_sizes(const mtx_model_desc* desc, int R, int shard_batch, mtx_sizes* out)
{
    if (!out) return fail(MTX_EINVAL, "out is NULL");
    Plan pl;
    int rc = make_plan(desc, R, shard_batch, pl);
    if (rc) return rc;
    out->n_params = pl.P;
    out->grad_stride = pl.ld;
    out->workspace_bytes = pl.ws_bytes;
    return MTX_OK;
}

}  // extern "C"

// Shared by mtx_init_model (workspace from the caller) and mtx_init_model_static (static_ws:
// the device's static array; bufs->workspace unused).
static int init_model(const mtx_model_desc* desc, int R, int shard_batch, uint64_t seed,
                      const mtx_buffers* bufs, void* stream, mtx_model** out, char* static_ws)
{
    if (!out) return fail(MTX_EINVAL, "out is NULL");
    *out = nullptr;
    if (!bufs) return fail(MTX_EINVAL, "bufs is NULL");
    Plan pl;
    int rc = make_plan(desc, R, shard_batch, pl);
    if (rc) return rc;
    if (!bufs->w || !bufs->v || !bufs->grads || !bufs->grad_avg ||
        (!static_ws && !bufs->workspace))
        return fail(MTX_EINVAL, "a model buffer is NULL");
    if (!aligned(bufs->w, 16) || !aligned(bufs->v, 16) || !aligned(bufs->grads, 16) ||
        !aligned(bufs->grad_avg, 16) || (!static_ws && !aligned(bufs->workspace, 256)))
        return fail(MTX_EINVAL, "model buffers must be 16-byte (workspace: 256-byte) aligned");
    if (static_ws) {
        if (pl.ws_bytes > kStaticScratchBytes)
            return fail(MTX_ENOMEM, "the network needs %zu bytes of workspace; the static "
                                    "workspace holds %zu (use mtx_init_model)",
                        pl.ws_bytes, kStaticScratchBytes);
        if (pl.jobs.size() > (size_t)kStaticMaxJobs)
            return fail(MTX_EUNSUPPORTED, "the network has %zu weight layouts to prepare; a "
                                          "static model takes at most %d (use mtx_init_model)",
                        pl.jobs.size(), kStaticMaxJobs);
    } else if (bufs->workspace_bytes < pl.ws_bytes) {
        return fail(MTX_ENOMEM, "workspace too small: %zu bytes given, %zu needed",
                    bufs->workspace_bytes, pl.ws_bytes);
    }
    void* wsp = static_ws ? static_cast<void*>(static_ws) : bufs->workspace;
    const size_t pb = pl.P * 4, gb = pl.ld * 4 * pl.R;
    if (overlap(bufs->w, pb, bufs->v, pb) || overlap(bufs->w, pb, bufs->grads, gb) ||
        overlap(bufs->w, pb, bufs->grad_avg, pb) || overlap(bufs->v, pb, bufs->grads, gb) ||
        overlap(bufs->v, pb, bufs->grad_avg, pb) || overlap(bufs->grads, gb, bufs->grad_avg, pb) ||
        overlap(wsp, pl.ws_bytes, bufs->w, pb) || overlap(wsp, pl.ws_bytes, bufs->v, pb) ||
        overlap(wsp, pl.ws_bytes, bufs->grads, gb) ||
        overlap(wsp, pl.ws_bytes, bufs->grad_avg, pb))
        return fail(MTX_EINVAL, "model buffers overlap");

    mtx_model* m = new (std::nothrow) mtx_model;
    if (!m) return fail(MTX_ENOMEM, "host allocation failed");
    m->pl = std::move(pl);
    m->w = bufs->w; m->v = bufs->v; m->grads = bufs->grads; m->gavg = bufs->grad_avg;
    m->ws = static_cast<char*>(wsp);
    m->static_ws = static_ws != nullptr;
    m->last_stream = static_cast<hipStream_t>(stream);
    // Measured on MI355X: running the weight gradients beside the data-gradient chain gains a
    // few percent when the step's matrix work is large (CIFAR-, AlexNet-sized steps) and loses
    // on small steps, whose kernels each fill the GPU on their own (LeNet).
    m->overlap = m->pl.gemm_flops >= 50e9;

    std::vector<float> w0;
    glorot_init_host(m->pl, seed, w0);
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e = hipStreamCreateWithFlags(&m->side, hipStreamNonBlocking);
    if (e != hipSuccess) m->side = nullptr;
    m->fork.assign(m->pl.n_wgrad, nullptr);
    for (size_t i = 0; i < m->fork.size() && e == hipSuccess; ++i)
        e = hipEventCreateWithFlags(&m->fork[i], hipEventDisableTiming);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&m->join, hipEventDisableTiming);
    if (e == hipSuccess) e = hipMemcpyAsync(m->w, w0.data(), pb, hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = hipMemsetAsync(m->v, 0, pb, s);
    // a static model sets up its part of the shared array at the start of every step instead
    if (!m->static_ws) {
        if (e == hipSuccess) e = hipMemsetAsync(m->ws + m->pl.sync_off, 0, kAlign, s);
        // the padded input's border and extra channels are never written by a step
        if (e == hipSuccess && m->pl.L.front().run)
            e = hipMemsetAsync(m->ws + m->pl.xin_off, 0, m->pl.xin_bytes, s);
        if (e == hipSuccess && !m->pl.jobs.empty())
            e = hipMemcpyAsync(m->ws + m->pl.jobs_off, m->pl.jobs.data(),
                               m->pl.jobs.size() * sizeof(PrepJob), hipMemcpyHostToDevice, s);
    }
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) {
        destroy_streams(m);
        delete m;
        return hip_fail(e, "mtx_init_model");
    }
    *out = m;
    return MTX_OK;
}

extern "C" {

int mtx_init_model(const mtx_model_desc* desc, int R, int shard_batch, uint64_t seed,
                   const mtx_buffers* bufs, void* stream, mtx_model** out)
{
    return init_model(desc, R, shard_batch, seed, bufs, stream, out, nullptr);
}

int mtx_init_model_static(const mtx_model_desc* desc, int R, int shard_batch, uint64_t seed,
                          const mtx_buffers* bufs, void* stream, mtx_model** out)
{
    if (out) *out = nullptr;
    if (bufs && (bufs->workspace || bufs->workspace_bytes))
        return fail(MTX_EINVAL, "a static model takes no workspace (workspace must be NULL, "
                                "workspace_bytes 0)");
    char* ws = nullptr;
    const int rc = static_scratch(&ws);
    if (rc) return rc;
    return init_model(desc, R, shard_batch, seed, bufs, stream, out, ws);
}

void mtx_free_model(mtx_model* m)
{
    if (!m) return;
    (void)hipStreamSynchronize(m->last_stream);
    if (m->side) (void)hipStreamSynchronize(m->side);
    if (m->upd) (void)hipStreamSynchronize(m->upd);
    m->graph.destroy();
    m->timer.destroy();
    destroy_streams(m);
    delete m;
}

int mtx_set_overlap(mtx_model* m, int enable)
{
    if (!m) return fail(MTX_EINVAL, "model is NULL");
    m->overlap = enable != 0;
    m->graph.reset();  // the captured launch sequence depends on it
    return MTX_OK;
}

int mtx_set_nonfinite_check(mtx_model* m, int enable)
{
    if (!m) return fail(MTX_EINVAL, "model is NULL");
    m->check_finite = enable != 0;
    m->graph.reset();  // the captured launch sequence depends on it
    return MTX_OK;
}

int mtx_set_fused_update(mtx_model* m, int enable)
{
    if (!m) return fail(MTX_EINVAL, "model is NULL");
    m->fuse_update = enable != 0;
    m->graph.reset();  // the captured launch sequence depends on it
    return MTX_OK;
}

int mtx_set_layerwise_update(mtx_model* m, int enable)
{
    if (!m) return fail(MTX_EINVAL, "model is NULL");
    // the third stream exists only while it is used: the box exposes few hardware queues, and
    // an idle extra stream can leave the weight-gradient stream sharing one with the caller's
    if (enable && !m->upd) {
        hipError_t e = hipStreamCreateWithFlags(&m->upd, hipStreamNonBlocking);
        if (e != hipSuccess) {
            m->upd = nullptr;
            return hip_fail(e, "mtx_set_layerwise_update");
        }
        m->wdone.assign(m->pl.n_wgrad, nullptr);
        m->ddone.assign(m->pl.n_wgrad, nullptr);
        for (size_t i = 0; i < m->wdone.size() && e == hipSuccess; ++i) {
            e = hipEventCreateWithFlags(&m->wdone[i], hipEventDisableTiming);
            if (e == hipSuccess) e = hipEventCreateWithFlags(&m->ddone[i], hipEventDisableTiming);
        }
        if (e == hipSuccess) e = hipEventCreateWithFlags(&m->upd_join, hipEventDisableTiming);
        if (e != hipSuccess) {
            release_update_stream(m);
            return hip_fail(e, "mtx_set_layerwise_update");
        }
    }
    if (!enable && m->upd) {
        (void)hipStreamSynchronize(m->upd);
        release_update_stream(m);
    }
    m->layerwise = enable != 0;
    m->graph.reset();  // the captured launch sequence depends on it
    return MTX_OK;
}

int mtx_set_timing(mtx_model* m, int enable)
{
    if (!m) return fail(MTX_EINVAL, "model is NULL");
    m->timer.on = enable != 0;
    return MTX_OK;
}

int mtx_get_timing(mtx_model* m, mtx_kernel_time* out, int capacity, int* count, int reset)
{
    if (!m || !count || capacity < 0 || (capacity > 0 && !out))
        return fail(MTX_EINVAL, "invalid arguments");
    HIP_TRY(m->timer.drain(), "read timing events");
    const int n = (int)m->timer.sites.size();
    *count = n;
    for (int i = 0; i < n && i < capacity; ++i) {
        const Timer::Site& st = m->timer.sites[i];
        std::memset(&out[i], 0, sizeof out[i]);
        std::snprintf(out[i].name, sizeof out[i].name, "%s", st.name.c_str());
        out[i].layer = st.layer;
        out[i].launches = (int)st.launches;
        out[i].total_ms = st.ms;
    }
    if (reset)
        for (auto& st : m->timer.sites) {
            st.ms = 0.0;
            st.launches = 0;
        }
    return MTX_OK;
}

// Enqueue the kernels of one step on stream s (eagerly, or into a capture).
// The average of the R shard gradients of parameters [off, off + len) fused with the model's
// update rule (Adam at step number m->opt_step, already advanced for this step).
static hipError_t update_slice(mtx_model* m, size_t off, size_t len, float lr, float momentum,
                               hipStream_t s, unsigned max_blocks)
{
    const Plan& pl = m->pl;
    if (m->opt == MTX_OPT_MOMENTUM)
        return average_update(m->grads + off, pl.R, len, pl.ld, m->w + off, m->v + off, lr,
                              momentum, m->gavg + off, true, s, max_blocks);
    AdaptParams p;
    p.w = m->w + off;
    p.s1 = m->v + off;
    p.s2 = m->opt == MTX_OPT_ADAM ? m->s2 + off : nullptr;
    p.avg = m->gavg + off;
    p.lr = lr;
    p.eps = m->eps;
    p.b1 = p.c1 = p.b2 = p.c2 = p.ib1 = p.ib2 = 0.0f;
    if (m->opt == MTX_OPT_ADAM) {
        const double t = (double)m->opt_step;
        p.b1 = m->b1;
        p.c1 = (float)(1.0 - (double)m->b1);
        p.b2 = m->b2;
        p.c2 = (float)(1.0 - (double)m->b2);
        p.ib1 = (float)(1.0 / (1.0 - std::pow((double)m->b1, t)));
        p.ib2 = (float)(1.0 / (1.0 - std::pow((double)m->b2, t)));
    }
    return average_adapt(m->grads + off, pl.R, len, pl.ld, m->opt == MTX_OPT_ADAM, p, s,
                         max_blocks);
}

static int enqueue_step(mtx_model* m, const float* x, const int32_t* labels, float lr,
                        float momentum, float* loss_out, hipStream_t s)
{
    const Plan& pl = m->pl;
    m->timer.cur = 0;
    m->launches.clear();
    const Dt dt = (Dt)pl.dt;
    const bool bf = pl.dt == MTX_BF16;
    char* ws = m->ws;
    if (m->static_ws) {
        // another static model may have used the array since this model's last step
        StaticSetup su{};
        su.njobs = (int)pl.jobs.size();
        for (int j = 0; j < su.njobs; ++j) su.jobs[j] = pl.jobs[j];
        su.dst_jobs = reinterpret_cast<PrepJob*>(ws + pl.jobs_off);
        su.sync = reinterpret_cast<unsigned*>(ws + pl.sync_off);
        const bool run0 = pl.L.front().run;
        su.zero = reinterpret_cast<uint4*>(ws + pl.xin_off);
        su.zero_vecs = run0 ? (pl.xin_bytes + 15) / 16 : 0;
        const unsigned blocks = (unsigned)std::min<unsigned long long>(
            1024ull, std::max<unsigned long long>(1ull, (su.zero_vecs + 255) / 256));
        HIP_TRY(launch_site(m, "static_setup", -1, s, [&] {
                    hipLaunchKernelGGL(static_setup_kernel, dim3(blocks), dim3(256), 0, s, su);
                    return hipGetLastError();
                }), "static workspace setup");
    }
    const size_t es = bf ? 2 : 4;
    const char* prep = ws + pl.prep_off;
    const void* x_in = pl.x_convert ? static_cast<const void*>(ws + pl.xin_off)
                                    : static_cast<const void*>(x);

    // ---- weights in the layouts the GEMMs read, input in the compute type and layout ----
    const LayerPlan& l0 = pl.L.front();
    // a direct first convolution carries the weight preparation in its own launch
    const bool prep_with_first = l0.direct && !pl.jobs.empty();
    if (!prep_with_first)
        HIP_TRY(launch_site(m, "prep_w", -1, s, [&] {
                    return prep_weights(dt, reinterpret_cast<const PrepJob*>(ws + pl.jobs_off),
                                        (int)pl.jobs.size(), pl.prep_blocks, m->w,
                                        ws + pl.prep_off, s);
                }), "weight preparation");
    if (pl.x_convert)
        HIP_TRY(launch_site(m, "prep_x", -1, s, [&] {
                    return l0.run ? to_nhwc_padded(dt, x, ws + pl.xin_off, pl.B, l0.c, l0.h, l0.w,
                                                   l0.p, l0.rg, s)
                                  : to_nhwc(dt, x, ws + pl.xin_off, pl.B, pl.x_c, pl.x_hw, s);
                }), "input conversion");
    auto fwd_w = [&](const LayerPlan& lp) { return prep + lp.fw_off * es; };
    auto bwd_w = [&](const LayerPlan& lp) { return prep + lp.bw_off * es; };
    float* partial = reinterpret_cast<float*>(ws + pl.partial_off);
    // ---- forward, all R shards at once (the weights are shared) ----
    const void* in = x_in;
    std::vector<char> add_done(pl.L.size(), 0);  // computed with the layer before it
    for (size_t l = 0; l < pl.L.size(); ++l) {
        const LayerPlan& lp = pl.L[l];
        void* out = ws + lp.act_off;
        const float* bias = m->w + lp.b_off;
        if (lp.kind == MTX_CONV && lp.direct) {
            ConvGeom g{pl.B, lp.c, lp.h, lp.w, lp.oc, lp.oh, lp.ow, lp.k, lp.s, lp.p, lp.g};
            FirstPoolFwd fp{};
            if (pl.pool_into_first) {
                fp.y = ws + pl.L[1].act_off;
                fp.argmax = reinterpret_cast<uint8_t*>(ws + pl.L[1].am_off);
                fp.k = pl.L[1].k;
            }
            FirstPrep pp{};
            if (prep_with_first) {
                pp.jobs = reinterpret_cast<const PrepJob*>(ws + pl.jobs_off);
                pp.njobs = (int)pl.jobs.size();
                pp.blocks = pl.prep_blocks;
                pp.w = m->w;
                pp.dst = ws + pl.prep_off;
            }
            HIP_TRY(launch_site(m, "fwd_direct", (int)l, s, [&] {
                        return first_conv_fwd(dt, g, in, m->w + lp.w_off, bias, out, lp.act_f32,
                                              lp.relu, s, fp, pp);
                    }), "first convolution forward (and the weight preparation)");
        } else if (lp.kind == MTX_CONV) {
            ConvGeom g{pl.B, lp.c, lp.h, lp.w, lp.oc, lp.oh, lp.ow, lp.k, lp.s, lp.p, lp.g};
            HIP_TRY(launch_site(m, "fwd", (int)l, s, [&] {
                        return lp.run ? conv_fwd_run(dt, g, lp.rg, in, fwd_w(lp), bias, out,
                                                     lp.act_f32, lp.relu, partial, s)
                                      : conv_fwd(dt, g, in, fwd_w(lp), bias, out, lp.act_f32,
                                                 lp.relu, partial, s);
                    }), "conv forward");
        } else if (lp.kind == MTX_FC) {
            HIP_TRY(launch_site(m, "fwd", (int)l, s, [&] {
                        return fc_fwd(dt, pl.B, (int)lp.in_elems, lp.oc, in, fwd_w(lp), bias, out,
                                      lp.act_f32, lp.relu, partial, s);
                    }), "fc forward");
        } else if (lp.kind == MTX_BN) {
            // A residual addition right after the batch normalisation is computed in the same
            // pass as its normalised output (which is still stored): the addition does not
            // read that output back.  A projection shortcut's convolution runs first.
            const LayerPlan* ap = l + 1 < pl.L.size() ? &pl.L[l + 1] : nullptr;
            const bool with_add = ap && (ap->kind == MTX_ADD || ap->kind == MTX_ADDP) &&
                                  !ap->act_f32 == !lp.act_f32;
            const void* other = nullptr;
            if (with_add && ap->kind == MTX_ADDP) {
                const LayerPlan& sp = pl.L[ap->src];
                HIP_TRY(launch_site(m, "fwd", (int)l + 1, s, [&] {
                            return conv_fwd(dt, proj_geom(*ap, sp, pl.B), ws + sp.act_off,
                                            fwd_w(*ap), m->w + ap->b_off, ws + ap->proj_off,
                                            ap->act_f32, false, partial, s);
                        }), "projection forward");
                other = ws + ap->proj_off;
            } else if (with_add) {
                other = ws + pl.L[ap->src].act_off;
            }
            if (with_add) add_done[l + 1] = 1;
            HIP_TRY(launch_site(m, "bn_fwd", (int)l, s, [&] {
                        return bn_fwd(dt, pl.R, pl.Nb, lp.h * lp.w, lp.c, in, out,
                                      m->w + lp.w_off, m->w + lp.b_off,
                                      reinterpret_cast<double*>(ws + pl.bn_part_off),
                                      reinterpret_cast<float*>(ws + lp.stat_off), lp.relu, s,
                                      other, with_add ? ws + ap->act_off : nullptr,
                                      with_add && ap->relu);
                    }), "batch norm forward");
        } else if (lp.kind == MTX_ADD) {
            if (!add_done[l])
                HIP_TRY(launch_site(m, "add_fwd", (int)l, s, [&] {
                            return add_fwd(dt, lp.out_elems * pl.B, in,
                                           ws + pl.L[lp.src].act_off, out, lp.relu, s);
                        }), "residual addition");
        } else if (lp.kind == MTX_ADDP) {
            // the projection (stored like a convolution's output), then the addition
            const LayerPlan& sp = pl.L[lp.src];
            void* pj = ws + lp.proj_off;
            if (!add_done[l]) {
                HIP_TRY(launch_site(m, "fwd", (int)l, s, [&] {
                            return conv_fwd(dt, proj_geom(lp, sp, pl.B), ws + sp.act_off,
                                            fwd_w(lp), bias, pj, lp.act_f32, false, partial, s);
                        }), "projection forward");
                HIP_TRY(launch_site(m, "add_fwd", (int)l, s, [&] {
                            return add_fwd(dt, lp.out_elems * pl.B, in, pj, out, lp.relu, s);
                        }), "projection addition");
            }
        } else if (!(l == 1 && pl.pool_into_first)) {  // else computed with layer 0
            HIP_TRY(launch_site(m, "pool_fwd", (int)l, s, [&] {
                        return pool_fwd(dt, pl.B, lp.c, lp.h, lp.w, lp.k, lp.s, !lp.nhwc, in, out,
                                        reinterpret_cast<uint8_t*>(ws + lp.am_off), s);
                    }), "pool forward");
        }
        in = out;
    }
    // ---- loss and its gradient (shard-mean loss: scale 1/Nb) ----
    const LayerPlan& last = pl.L.back();
    float* block_sums = reinterpret_cast<float*>(ws + pl.loss_off);
    unsigned* sync = reinterpret_cast<unsigned*>(ws + pl.sync_off);
    HIP_TRY(launch_site(m, "softmax_xent", -1, s, [&] {
                return softmax_xent(dt, pl.B, last.oc, pl.Nb,
                                    reinterpret_cast<const float*>(ws + last.act_off), labels,
                                    ws + last.dy_off, block_sums, sync, loss_out, s);
            }), "softmax cross-entropy");

    // ---- backward in reverse layer order; weight gradients per shard into grads[r] ----
    // The data gradients form a chain on stream s.  A weight gradient needs only its layer's
    // output gradient and input, so (unless kernels are being timed) it runs on the second
    // stream, forked after its output gradient is written and joined before the update.
    const bool overlap = m->overlap && !m->timer.on;
    const bool layerwise = m->layerwise && m->upd && !m->timer.on && !m->check_finite;
    float* partial_w = overlap ? reinterpret_cast<float*>(ws + pl.partial_w_off) : partial;
    const long long ld = (long long)pl.ld;
    int nfork = 0, nlayer = 0;
    // Large fully connected layers (AlexNet's three) take the average + update of their own
    // parameters in their weight-gradient launch, with the momentum rule and without the
    // layer-wise option: the R shard rows are summed while they are written instead of being
    // read back at the end (AlexNet: 1.2 GB less traffic), and the update runs beside the rest of
    // the backward pass.  The average + update at the end covers the other parameters, in
    // contiguous ranges (`rest`).
    std::vector<char> fused(pl.L.size(), 0);
    std::vector<std::pair<size_t, size_t>> rest;
    {
        const bool can = m->fuse_update && m->opt == MTX_OPT_MOMENTUM && !layerwise &&
                         !m->check_finite;
        size_t beg = 0;
        for (size_t l = 0; l < pl.L.size(); ++l) {
            const LayerPlan& lp = pl.L[l];
            fused[l] = can && lp.kind == MTX_FC && (int)l >= pl.first_param &&
                       fc_wgrad_update_ok(dt, pl.Nb, pl.R, (int)lp.in_elems, lp.oc);
            if (!fused[l]) continue;
            if (lp.w_off > beg) rest.emplace_back(beg, lp.w_off - beg);
            beg = lp.b_off + lp.b_len;
        }
        if (pl.P > beg) rest.emplace_back(beg, pl.P - beg);
    }
    for (int l = (int)pl.L.size() - 1; l >= pl.first_param && l >= 0; --l) {
        const LayerPlan& lp = pl.L[l];
        const void* in_l = l == 0 ? x_in : static_cast<const void*>(ws + pl.L[l - 1].act_off);
        const void* dy = ws + lp.dy_off;
        void* dx = lp.need_dx ? ws + pl.L[l - 1].dy_off : nullptr;
        const void* mask = (l > 0 && pl.L[l - 1].relu) ? ws + pl.L[l - 1].act_off : nullptr;
        const bool mask_f32 = l > 0 && pl.L[l - 1].act_f32;
        hipStream_t sw = s;
        // The first parameter layer has no data gradient to run beside: its weight gradient runs
        // on the caller's stream, beside the weight gradients still running on the second stream
        // (measured on the AlexNet step: conv1's weight gradient no longer trails the others).
        const bool side = lp.w_len && overlap && lp.kind != MTX_BN && l != pl.first_param;
        float* part_wg = side ? partial_w : partial;
        if (side) {
            HIP_TRY(hipEventRecord(m->fork[nfork], s), "fork");
            HIP_TRY(hipStreamWaitEvent(m->side, m->fork[nfork], 0), "fork");
            ++nfork;
            sw = m->side;
        }
        if (lp.kind == MTX_CONV && lp.direct) {
            ConvGeom gs{pl.Nb, lp.c, lp.h, lp.w, lp.oc, lp.oh, lp.ow, lp.k, lp.s, lp.p, lp.g};
            FirstPool fp{};
            if (pl.pool_into_first) {
                const LayerPlan& p1 = pl.L[1];
                fp.dy = ws + p1.dy_off;
                fp.argmax = reinterpret_cast<const uint8_t*>(ws + p1.am_off);
                fp.gate = lp.relu ? ws + p1.act_off : nullptr;
                fp.k = p1.k;
            }
            HIP_TRY(launch_site(m, "wgrad_direct", l, sw, [&] {
                        return first_conv_wgrad(dt, gs, pl.R, in_l, dy,
                                                reinterpret_cast<float*>(ws + pl.first_part_off),
                                                m->grads, ld, (long long)lp.w_off,
                                                (long long)lp.b_off, sw, fp);
                    }), "first convolution weight gradient");
        } else if (lp.kind == MTX_CONV) {
            ConvGeom gs{pl.Nb, lp.c, lp.h, lp.w, lp.oc, lp.oh, lp.ow, lp.k, lp.s, lp.p, lp.g};
            HIP_TRY(launch_site(m, "wgrad", l, sw, [&] {
                        return lp.run ? conv_wgrad_run(dt, gs, lp.rg, pl.R, in_l, dy, m->grads, ld,
                                                       (long long)lp.w_off, (long long)lp.b_off,
                                                       part_wg, sw)
                                      : conv_wgrad(dt, gs, pl.R, in_l, dy, m->grads, ld,
                                                   (long long)lp.w_off, (long long)lp.b_off,
                                                   part_wg, sw);
                    }), "conv weight gradient");
            if (lp.need_dx) {
                ConvGeom g{pl.B, lp.c, lp.h, lp.w, lp.oc, lp.oh, lp.ow, lp.k, lp.s, lp.p, lp.g};
                float* col = reinterpret_cast<float*>(ws + pl.col_off);
                HIP_TRY(launch_site(m, "dgrad", l, s, [&] {
                            if (lp.dgrad_fused)
                                return conv_dgrad_fused(g, static_cast<const float*>(dy),
                                                        m->w + lp.w_off, static_cast<float*>(dx),
                                                        mask, mask_f32, s);
                            return lp.dgrad_col
                                       ? conv_dgrad_col(dt, g, dy, bwd_w(lp), dx, mask, mask_f32,
                                                        col, partial, s)
                                       : conv_dgrad(dt, g, dy, bwd_w(lp), dx, mask, mask_f32,
                                                    partial, s);
                        }), "conv data gradient");
            }
        } else if (lp.kind == MTX_FC && fused[l]) {
            HIP_TRY(launch_site(m, "wgrad_update", l, sw, [&] {
                        return fc_wgrad_update(dt, pl.Nb, pl.R, (int)lp.in_elems, lp.oc,
                                               lp.perm_c, lp.perm_hw, in_l, dy, m->grads, ld,
                                               (long long)lp.w_off, (long long)lp.b_off, m->w,
                                               m->v, m->gavg, lr, momentum, sw);
                    }), "fc weight gradient + average + update");
            if (lp.need_dx)
                HIP_TRY(launch_site(m, "dgrad", l, s, [&] {
                            return fc_dgrad(dt, pl.B, (int)lp.in_elems, lp.oc, dy, bwd_w(lp), dx,
                                            mask, mask_f32, partial, s);
                        }), "fc data gradient");
        } else if (lp.kind == MTX_FC) {
            HIP_TRY(launch_site(m, "wgrad", l, sw, [&] {
                        return fc_wgrad(dt, pl.Nb, pl.R, (int)lp.in_elems, lp.oc, lp.perm_c,
                                        lp.perm_hw, in_l, dy, m->grads, ld, (long long)lp.w_off,
                                        (long long)lp.b_off, part_wg, sw);
                    }), "fc weight gradient");
            if (lp.need_dx)
                HIP_TRY(launch_site(m, "dgrad", l, s, [&] {
                            return fc_dgrad(dt, pl.B, (int)lp.in_elems, lp.oc, dy, bwd_w(lp), dx,
                                            mask, mask_f32, partial, s);
                        }), "fc data gradient");
        } else if (lp.kind == MTX_BN) {
            HIP_TRY(launch_site(m, "bn_bwd", l, s, [&] {
                        return bn_bwd(dt, pl.R, pl.Nb, lp.h * lp.w, lp.c, in_l, dy, dx, mask,
                                      mask_f32, reinterpret_cast<const float*>(ws + lp.stat_off),
                                      reinterpret_cast<double*>(ws + pl.bn_part_off),
                                      reinterpret_cast<float*>(ws + pl.bn_coef_off), m->grads, ld,
                                      (long long)lp.w_off, (long long)lp.b_off, s);
                    }), "batch norm backward");
        } else if (lp.kind == MTX_ADD) {
            // the previous layer's share: dy (times its ReLU mask), unless it reads dy itself;
            // the source's share is added from dy when the source's gradient is written
            if (dx && !lp.dy_shared)
                HIP_TRY(launch_site(m, "add_bwd", l, s, [&] {
                            return add_bwd(dt, lp.out_elems * pl.B, dy, dx, mask, mask_f32,
                                           nullptr, nullptr, false, s);
                        }), "residual backward");
        } else if (lp.kind == MTX_ADDP) {
            // the previous layer's gradient is dy (times its ReLU mask); the projection's weight
            // gradient (per shard, on the weight-gradient stream) and its data gradient, which
            // becomes the gradient kept for the source (times the source's ReLU mask)
            const LayerPlan& sp = pl.L[lp.src];
            HIP_TRY(launch_site(m, "wgrad", l, sw, [&] {
                        return conv_wgrad(dt, proj_geom(lp, sp, pl.Nb), pl.R, ws + sp.act_off, dy,
                                          m->grads, ld, (long long)lp.w_off, (long long)lp.b_off,
                                          part_wg, sw);
                    }), "projection weight gradient");
            if (dx && !lp.dy_shared)
                HIP_TRY(launch_site(m, "add_bwd", l, s, [&] {
                            return add_bwd(dt, lp.out_elems * pl.B, dy, dx, mask, mask_f32,
                                           nullptr, nullptr, false, s);
                        }), "projection addition backward");
            if (lp.skip_off != kNone)
                HIP_TRY(launch_site(m, "dgrad", l, s, [&] {
                            const ConvGeom gp = proj_geom(lp, sp, pl.B);
                            const void* smask = sp.relu ? ws + sp.act_off : nullptr;
                            return lp.dgrad_col
                                       ? conv_dgrad_col(dt, gp, dy, bwd_w(lp), ws + lp.skip_off,
                                                        smask, sp.act_f32,
                                                        reinterpret_cast<float*>(ws + pl.col_off),
                                                        partial, s)
                                       : conv_dgrad(dt, gp, dy, bwd_w(lp), ws + lp.skip_off,
                                                    smask, sp.act_f32, partial, s);
                        }), "projection data gradient");
        } else if (lp.need_dx && !(l == 1 && pl.pool_into_first)) {
            HIP_TRY(launch_site(m, "pool_bwd", l, s, [&] {
                        return pool_bwd(dt, pl.B, lp.c, lp.h, lp.w, lp.k, lp.s, !lp.nhwc,
                                        reinterpret_cast<const uint8_t*>(ws + lp.am_off), dy, dx,
                                        mask ? ws + lp.act_off : nullptr, s);
                    }), "pool backward");
        }
        // The output gradient of layer l - 1 is now written; if a residual addition also read
        // that layer's output, add its share (before the layer's own weight gradient is forked
        // off on the next iteration): an identity addition's output gradient, times the ReLU
        // mask of layer l - 1, or a projection's data gradient, which has the mask applied.
        if (lp.need_dx)
            for (size_t a2 = (size_t)l + 1; a2 < pl.L.size(); ++a2) {
                const LayerPlan& ap = pl.L[a2];
                if (ap.src != l - 1 || (ap.kind != MTX_ADD && ap.kind != MTX_ADDP) ||
                    (ap.kind == MTX_ADDP && ap.skip_off == kNone))
                    continue;
                const LayerPlan& sp = pl.L[l - 1];
                const bool ident = ap.kind == MTX_ADD;
                HIP_TRY(launch_site(m, "skip_add", l - 1, s, [&] {
                            return skip_add(dt, sp.out_elems * pl.B, ws + sp.dy_off,
                                            ws + (ident ? ap.dy_off : ap.skip_off),
                                            ident && sp.relu ? ws + sp.act_off : nullptr,
                                            sp.act_f32, s);
                        }), "residual gradient");
            }
        // Layer-wise averaging (the paper issues one reduction per layer, in layer order): this
        // layer's parameters are averaged and updated on the third stream as soon as its R
        // shard gradients are written, beside the rest of the backward pass.  The update waits
        // for the layer's weight gradients (on sw) and for every kernel enqueued so far on s,
        // among them the layer's own data gradient, which may read its master weights (the
        // fused small-image data gradient does); later kernels read only other layers' weights
        // or the prepared copies.
        if (lp.w_len && layerwise) {
            HIP_TRY(hipEventRecord(m->wdone[nlayer], sw), "layer gradients done");
            HIP_TRY(hipStreamWaitEvent(m->upd, m->wdone[nlayer], 0), "layer gradients done");
            if (sw != s) {
                HIP_TRY(hipEventRecord(m->ddone[nlayer], s), "layer data gradient done");
                HIP_TRY(hipStreamWaitEvent(m->upd, m->ddone[nlayer], 0), "layer data gradient done");
            }
            ++nlayer;
            const size_t off = lp.w_off, len = lp.w_len + lp.b_len;
            HIP_TRY(launch_site(m, "avg_update", l, m->upd, [&] {
                        return update_slice(m, off, len, lr, momentum, m->upd,
                                            kLayerUpdateBlocks);
                    }), "layer average + update");
        }
    }
    if (nfork) {
        HIP_TRY(hipEventRecord(m->join, m->side), "join");
        HIP_TRY(hipStreamWaitEvent(s, m->join, 0), "join");
    }
    if (nlayer) {
        HIP_TRY(hipEventRecord(m->upd_join, m->upd), "join");
        HIP_TRY(hipStreamWaitEvent(s, m->upd_join, 0), "join");
        return MTX_OK;
    }
    // ---- average of the R shard gradients fused with the optimizer step ----
    if (m->check_finite) {
        // the average first, with a flag for a non-finite value; then the momentum update from
        // the stored average (g = avg / 1: the same values as the fused pass), which does
        // nothing while the flag is set
        int* flag = reinterpret_cast<int*>(ws + pl.sync_off + 64);
        HIP_TRY(set_flag(flag, 0, s), "non-finite flag");
        HIP_TRY(launch_site(m, "avg_update", -1, s, [&] {
                    return average_update(m->grads, pl.R, pl.P, pl.ld, m->w, m->v, lr, momentum,
                                          m->gavg, false, s, 0, nullptr, flag);
                }), "average");
        HIP_TRY(launch_site(m, "avg_update", -1, s, [&] {
                    return average_update(m->gavg, 1, pl.P, pl.ld, m->w, m->v, lr, momentum,
                                          nullptr, true, s, 0, flag, nullptr);
                }), "update");
        return MTX_OK;
    }
    for (const auto& rg : rest)
        HIP_TRY(launch_site(m, "avg_update", -1, s, [&] {
                    return update_slice(m, rg.first, rg.second, lr, momentum, s, 0);
                }), "average + update");
    return MTX_OK;
}

// Capture one step into a new executable graph; on any failure the capture is abandoned and
// the caller falls back to enqueuing the step directly.
static bool capture_step(mtx_model* m, const float* x, const int32_t* labels, float lr,
                         float momentum, float* loss_out)
{
    GraphCache& gc = m->graph;
    gc.reset();
    if (!gc.capture_stream &&
        hipStreamCreateWithFlags(&gc.capture_stream, hipStreamNonBlocking) != hipSuccess) {
        gc.capture_stream = nullptr;
        return false;
    }
    if (hipStreamBeginCapture(gc.capture_stream, hipStreamCaptureModeThreadLocal) != hipSuccess)
        return false;
    const std::string saved = g_err;
    const int rc = enqueue_step(m, x, labels, lr, momentum, loss_out, gc.capture_stream);
    hipGraph_t graph = nullptr;
    const hipError_t e = hipStreamEndCapture(gc.capture_stream, &graph);
    g_err = saved;
    if (rc != MTX_OK || e != hipSuccess || !graph) {
        if (graph) (void)hipGraphDestroy(graph);
        (void)hipGetLastError();
        return false;
    }
    hipGraphExec_t exec = nullptr;
    const hipError_t ei = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
    (void)hipGraphDestroy(graph);
    if (ei != hipSuccess) {
        (void)hipGetLastError();
        return false;
    }
    gc.exec = exec;
    gc.x = x; gc.labels = labels; gc.lr = lr; gc.mu = momentum; gc.loss = loss_out;
    return true;
}

static int step_dispatch(mtx_model* m, const float* x, const int32_t* labels, float lr,
                         float momentum, float* loss_out, hipStream_t s, bool caller_capturing);

int mtx_train_step(mtx_model* m, const float* x, const int32_t* labels, float lr,
                   float momentum, float* loss_out, void* stream)
{
    if (!m) return fail(MTX_EINVAL, "model is NULL");
    if (!x || !labels) return fail(MTX_EINVAL, "x and labels must not be NULL");
    if (!aligned(x, 16) || !aligned(labels, 4) || (loss_out && !aligned(loss_out, 4)))
        return fail(MTX_EINVAL, "x must be 16-byte aligned, labels and loss_out 4-byte aligned");
    if (!std::isfinite(lr) || !std::isfinite(momentum))
        return fail(MTX_EINVAL, "lr and momentum must be finite");
    hipStream_t s = static_cast<hipStream_t>(stream);
    GraphCache& gc = m->graph;
    hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
    const bool caller_capturing =
        hipStreamIsCapturing(s, &cap) == hipSuccess && cap != hipStreamCaptureStatusNone;
    (void)hipGetLastError();
    if (m->check_finite && (m->opt != MTX_OPT_MOMENTUM || caller_capturing))
        return fail(MTX_EUNSUPPORTED, "the non-finite check needs the momentum rule and a stream "
                                      "that is not being captured");
    m->last_stream = s;
    ++m->opt_step;
    if (m->check_finite) {
        const int rc = step_dispatch(m, x, labels, lr, momentum, loss_out, s, caller_capturing);
        if (rc != MTX_OK) return rc;
        int flag = 0;
        HIP_TRY(hipMemcpyAsync(&flag, m->ws + m->pl.sync_off + 64, sizeof flag,
                               hipMemcpyDeviceToHost, s), "non-finite flag");
        HIP_TRY(hipStreamSynchronize(s), "non-finite flag");
        if (flag) return fail(MTX_ENONFINITE, "the gradient average is not finite: w and v kept");
        return MTX_OK;
    }
    return step_dispatch(m, x, labels, lr, momentum, loss_out, s, caller_capturing);
}

// The step on stream s: replayed from the model's graph, captured into it, or enqueued directly.
static int step_dispatch(mtx_model* m, const float* x, const int32_t* labels, float lr,
                         float momentum, float* loss_out, hipStream_t s, bool caller_capturing)
{
    GraphCache& gc = m->graph;
    // Adam's bias correction changes every step, so its steps are not replayed from a graph
    if (gc.enabled && !m->timer.on && !caller_capturing && m->opt != MTX_OPT_ADAM &&
        gc.misses < GraphCache::kMaxMisses) {
        if (gc.matches(x, labels, lr, momentum, loss_out)) {
            gc.misses = 0;
            HIP_TRY(hipGraphLaunch(gc.exec, s), "graph launch");
            return MTX_OK;
        }
        gc.misses += 1;
        if (capture_step(m, x, labels, lr, momentum, loss_out)) {
            HIP_TRY(hipGraphLaunch(gc.exec, s), "graph launch");
            return MTX_OK;
        }
        gc.misses = GraphCache::kMaxMisses;  // capture is not possible here: stay eager
    }
    return enqueue_step(m, x, labels, lr, momentum, loss_out, s);
}

int mtx_get_launches(const mtx_model* m, mtx_launch_info* out, int capacity, int* count)
{
    if (!m || !count || capacity < 0 || (capacity > 0 && !out))
        return fail(MTX_EINVAL, "invalid arguments");
    const int n = (int)m->launches.size();
    *count = n;
    for (int i = 0; i < n && i < capacity; ++i) out[i] = m->launches[i];
    return MTX_OK;
}

int mtx_set_optimizer(mtx_model* m, int kind, float beta1, float beta2, float eps, float* s2)
{
    if (!m) return fail(MTX_EINVAL, "model is NULL");
    if (kind != MTX_OPT_MOMENTUM && kind != MTX_OPT_ADAM && kind != MTX_OPT_ADAGRAD)
        return fail(MTX_EINVAL, "unknown optimizer %d", kind);
    if (kind != MTX_OPT_MOMENTUM && (!std::isfinite(eps) || eps < 0.0f))
        return fail(MTX_EINVAL, "eps must be finite and >= 0");
    if (kind == MTX_OPT_ADAM) {
        if (!(beta1 >= 0.0f && beta1 < 1.0f) || !(beta2 >= 0.0f && beta2 < 1.0f))
            return fail(MTX_EINVAL, "beta1 and beta2 must lie in [0, 1)");
        if (!s2 || !aligned(s2, 16))
            return fail(MTX_EINVAL, "Adam needs a 16-byte aligned second-moment buffer");
        const size_t nb = m->pl.P * 4;
        if (overlap(s2, nb, m->w, nb) || overlap(s2, nb, m->v, nb) ||
            overlap(s2, nb, m->gavg, nb) || overlap(s2, nb, m->grads, m->pl.ld * m->pl.R * 4))
            return fail(MTX_EINVAL, "the second-moment buffer overlaps the model's buffers");
    }
    m->opt = kind;
    m->b1 = beta1;
    m->b2 = beta2;
    m->eps = eps;
    m->s2 = kind == MTX_OPT_ADAM ? s2 : nullptr;
    m->opt_step = 0;
    m->graph.reset();  // a recorded step holds the previous update rule
    return MTX_OK;
}

int mtx_set_graph_replay(mtx_model* m, int enable)
{
    if (!m) return fail(MTX_EINVAL, "model is NULL");
    m->graph.enabled = enable != 0;
    m->graph.misses = 0;
    if (!enable) m->graph.reset();
    return MTX_OK;
}

static int check_avg_args(const float* grads, int R, size_t n, size_t ld, const float* out)
{
    if (!grads || !out) return fail(MTX_EINVAL, "grads and the output must not be NULL");
    if (R < 1) return fail(MTX_EINVAL, "R must be >= 1 (got %d)", R);
    if (n < 1) return fail(MTX_EINVAL, "n must be >= 1");
    if (ld < n) return fail(MTX_EINVAL, "ld must be >= n");
    if (!aligned(grads, 4) || !aligned(out, 4)) return fail(MTX_EINVAL, "pointers must be 4-byte aligned");
    if ((unsigned long long)ld * R > (1ull << 62)) return fail(MTX_EINVAL, "sizes overflow");
    return MTX_OK;
}

int mtx_average_grads(const float* grads, int R, size_t n, size_t ld, float* avg, void* stream)
{
    int rc = check_avg_args(grads, R, n, ld, avg);
    if (rc) return rc;
    const size_t gb = ((size_t)(R - 1) * ld + n) * 4;
    if (overlap(grads, gb, avg, n * 4)) return fail(MTX_EINVAL, "avg overlaps grads");
    HIP_TRY(average_update(grads, R, n, ld, nullptr, nullptr, 0.f, 0.f, avg, false,
                           static_cast<hipStream_t>(stream)), "mtx_average_grads");
    return MTX_OK;
}

int mtx_sgd_update(float* w, float* v, const float* grads, int R, size_t n, size_t ld, float lr,
                   float momentum, float* avg_out, void* stream)
{
    int rc = check_avg_args(grads, R, n, ld, w);
    if (rc) return rc;
    if (!std::isfinite(lr) || !std::isfinite(momentum))
        return fail(MTX_EINVAL, "lr and momentum must be finite");
    if (momentum != 0.0f && !v) return fail(MTX_EINVAL, "v must not be NULL when momentum != 0");
    if ((v && !aligned(v, 4)) || (avg_out && !aligned(avg_out, 4)))
        return fail(MTX_EINVAL, "pointers must be 4-byte aligned");
    const size_t gb = ((size_t)(R - 1) * ld + n) * 4, nb = n * 4;
    if (overlap(grads, gb, w, nb) || (v && overlap(grads, gb, v, nb)) ||
        (avg_out && overlap(grads, gb, avg_out, nb)) || (v && overlap(w, nb, v, nb)) ||
        (avg_out && overlap(w, nb, avg_out, nb)) || (v && avg_out && overlap(v, nb, avg_out, nb)))
        return fail(MTX_EINVAL, "w, v, avg_out and grads must not overlap");
    HIP_TRY(average_update(grads, R, n, ld, w, momentum != 0.0f ? v : nullptr, lr, momentum, avg_out,
                           true, static_cast<hipStream_t>(stream)), "mtx_sgd_update");
    return MTX_OK;
}

// Pairwise overlap test over the non-null buffers of an update (grads spans gb bytes, every
// other buffer n floats).
static bool any_overlap(const float* grads, size_t gb, size_t nb, std::initializer_list<const float*> bufs)
{
    std::vector<const float*> b;
    for (const float* p : bufs)
        if (p) b.push_back(p);
    for (size_t i = 0; i < b.size(); ++i) {
        if (overlap(grads, gb, b[i], nb)) return true;
        for (size_t j = i + 1; j < b.size(); ++j)
            if (overlap(b[i], nb, b[j], nb)) return true;
    }
    return false;
}

int mtx_adam_update(float* w, float* m, float* v, const float* grads, int R, size_t n, size_t ld,
                    float lr, float beta1, float beta2, float eps, long long step, float* avg_out,
                    void* stream)
{
    int rc = check_avg_args(grads, R, n, ld, w);
    if (rc) return rc;
    if (!m || !v) return fail(MTX_EINVAL, "m and v must not be NULL");
    if (!aligned(m, 4) || !aligned(v, 4) || (avg_out && !aligned(avg_out, 4)))
        return fail(MTX_EINVAL, "pointers must be 4-byte aligned");
    if (!std::isfinite(lr) || !std::isfinite(eps) || eps < 0.0f)
        return fail(MTX_EINVAL, "lr must be finite and eps finite and >= 0");
    if (!(beta1 >= 0.0f && beta1 < 1.0f) || !(beta2 >= 0.0f && beta2 < 1.0f))
        return fail(MTX_EINVAL, "beta1 and beta2 must lie in [0, 1)");
    if (step < 1) return fail(MTX_EINVAL, "step must be >= 1 (got %lld)", step);
    const size_t gb = ((size_t)(R - 1) * ld + n) * 4, nb = n * 4;
    if (any_overlap(grads, gb, nb, {w, m, v, avg_out}))
        return fail(MTX_EINVAL, "w, m, v, avg_out and grads must not overlap");
    AdaptParams p;
    p.w = w;
    p.s1 = m;
    p.s2 = v;
    p.avg = avg_out;
    p.lr = lr;
    p.b1 = beta1;
    p.c1 = (float)(1.0 - (double)beta1);
    p.b2 = beta2;
    p.c2 = (float)(1.0 - (double)beta2);
    p.ib1 = (float)(1.0 / (1.0 - std::pow((double)beta1, (double)step)));
    p.ib2 = (float)(1.0 / (1.0 - std::pow((double)beta2, (double)step)));
    p.eps = eps;
    HIP_TRY(average_adapt(grads, R, n, ld, true, p, static_cast<hipStream_t>(stream)),
            "mtx_adam_update");
    return MTX_OK;
}

int mtx_adagrad_update(float* w, float* acc, const float* grads, int R, size_t n, size_t ld,
                       float lr, float eps, float* avg_out, void* stream)
{
    int rc = check_avg_args(grads, R, n, ld, w);
    if (rc) return rc;
    if (!acc) return fail(MTX_EINVAL, "acc must not be NULL");
    if (!aligned(acc, 4) || (avg_out && !aligned(avg_out, 4)))
        return fail(MTX_EINVAL, "pointers must be 4-byte aligned");
    if (!std::isfinite(lr) || !std::isfinite(eps) || eps < 0.0f)
        return fail(MTX_EINVAL, "lr must be finite and eps finite and >= 0");
    const size_t gb = ((size_t)(R - 1) * ld + n) * 4, nb = n * 4;
    if (any_overlap(grads, gb, nb, {w, acc, avg_out}))
        return fail(MTX_EINVAL, "w, acc, avg_out and grads must not overlap");
    AdaptParams p;
    p.w = w;
    p.s1 = acc;
    p.s2 = nullptr;
    p.avg = avg_out;
    p.lr = lr;
    p.b1 = p.c1 = p.b2 = p.c2 = p.ib1 = p.ib2 = 0.0f;
    p.eps = eps;
    HIP_TRY(average_adapt(grads, R, n, ld, false, p, static_cast<hipStream_t>(stream)),
            "mtx_adagrad_update");
    return MTX_OK;
}

int mtx_get_params(const mtx_model* m, float* w_host, float* v_host)
{
    if (!m || !w_host) return fail(MTX_EINVAL, "model and w_host must not be NULL");
    HIP_TRY(hipStreamSynchronize(m->last_stream), "synchronise");
    HIP_TRY(hipMemcpy(w_host, m->w, m->pl.P * 4, hipMemcpyDeviceToHost), "copy w");
    if (v_host) HIP_TRY(hipMemcpy(v_host, m->v, m->pl.P * 4, hipMemcpyDeviceToHost), "copy v");
    return MTX_OK;
}

int mtx_set_params(mtx_model* m, const float* w_host, const float* v_host)
{
    if (!m || !w_host) return fail(MTX_EINVAL, "model and w_host must not be NULL");
    HIP_TRY(hipStreamSynchronize(m->last_stream), "synchronise");
    HIP_TRY(hipMemcpy(m->w, w_host, m->pl.P * 4, hipMemcpyHostToDevice), "copy w");
    if (v_host) HIP_TRY(hipMemcpy(m->v, v_host, m->pl.P * 4, hipMemcpyHostToDevice), "copy v");
    return MTX_OK;
}

// Host copy of a stored layer output in NCHW order (NHWC on the device for convolution and
// pooling layers), as fp32.
int mtx_get_layer_output(const mtx_model* m, int layer, float* dst_host, size_t n)
{
    if (!m || !dst_host) return fail(MTX_EINVAL, "model and dst_host must not be NULL");
    if (layer < 0 || layer >= (int)m->pl.L.size()) return fail(MTX_EINVAL, "layer out of range");
    const LayerPlan& lp = m->pl.L[layer];
    const size_t cnt = lp.out_elems * m->pl.B;
    if (n < cnt) return fail(MTX_EINVAL, "dst_host holds %zu elements, %zu needed", n, cnt);
    HIP_TRY(hipStreamSynchronize(m->last_stream), "synchronise");
    std::vector<float> dev;
    std::vector<uint16_t> tmp;
    try {
        dev.resize(cnt);
        if (!lp.act_f32) tmp.resize(cnt);
    } catch (...) {
        return fail(MTX_ENOMEM, "host allocation failed");
    }
    if (lp.act_f32) {
        HIP_TRY(hipMemcpy(dev.data(), m->ws + lp.act_off, cnt * 4, hipMemcpyDeviceToHost), "copy");
    } else {
        HIP_TRY(hipMemcpy(tmp.data(), m->ws + lp.act_off, cnt * 2, hipMemcpyDeviceToHost), "copy");
        for (size_t i = 0; i < cnt; ++i) {
            const uint32_t u = static_cast<uint32_t>(tmp[i]) << 16;
            std::memcpy(&dev[i], &u, 4);
        }
    }
    if (!lp.nhwc) {
        std::memcpy(dst_host, dev.data(), cnt * 4);
        return MTX_OK;
    }
    const size_t C = lp.oc, HW = (size_t)lp.oh * lp.ow;
    for (size_t b = 0; b < (size_t)m->pl.B; ++b)
        for (size_t hw = 0; hw < HW; ++hw)
            for (size_t c = 0; c < C; ++c)
                dst_host[(b * C + c) * HW + hw] = dev[(b * HW + hw) * C + c];
    return MTX_OK;
}

// Host copy of a max-pooling layer's window decisions in NCHW order.
int mtx_get_pool_argmax(const mtx_model* m, int layer, uint8_t* dst_host, size_t n)
{
    if (!m || !dst_host) return fail(MTX_EINVAL, "model and dst_host must not be NULL");
    if (layer < 0 || layer >= (int)m->pl.L.size() || m->pl.L[layer].kind != MTX_MAXPOOL)
        return fail(MTX_EINVAL, "layer %d is not a max-pooling layer", layer);
    const LayerPlan& lp = m->pl.L[layer];
    const size_t cnt = lp.out_elems * m->pl.B;
    if (n < cnt) return fail(MTX_EINVAL, "dst_host holds %zu elements, %zu needed", n, cnt);
    HIP_TRY(hipStreamSynchronize(m->last_stream), "synchronise");
    std::vector<uint8_t> dev;
    try {
        dev.resize(cnt);
    } catch (...) {
        return fail(MTX_ENOMEM, "host allocation failed");
    }
    HIP_TRY(hipMemcpy(dev.data(), m->ws + lp.am_off, cnt, hipMemcpyDeviceToHost), "copy");
    if (!lp.nhwc) {
        std::memcpy(dst_host, dev.data(), cnt);
        return MTX_OK;
    }
    const size_t C = lp.oc, HW = (size_t)lp.oh * lp.ow;
    for (size_t b = 0; b < (size_t)m->pl.B; ++b)
        for (size_t hw = 0; hw < HW; ++hw)
            for (size_t c = 0; c < C; ++c)
                dst_host[(b * C + c) * HW + hw] = dev[(b * HW + hw) * C + c];
    return MTX_OK;
}

}  // extern "C"
