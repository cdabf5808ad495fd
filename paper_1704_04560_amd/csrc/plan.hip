// Launch planning for the implicit GEMMs (host only), shared by the workspace sizing in
// api.hip and by the launches, so that both always agree.
#include <algorithm>

#include "internal.h"

namespace mtx {

FastDiv make_fastdiv(unsigned d)
{
    FastDiv f{};
    if (d == 0) d = 1;
    unsigned s = 0;
    while ((1ull << s) < d) ++s;
    f.m = (unsigned)((((1ull << 32) * ((1ull << s) - d)) / d) + 1);
    f.s = s;
    return f;
}

int vec_elems(int dt) { return dt == DT_F32 ? 4 : 8; }

static long long cdiv(long long a, long long b) { return (a + b - 1) / b; }

// Tile: the largest of 128x128, 64x128, 64x64, 32x128, 32x64 (rows x columns) that gives at
// least two blocks per compute unit, or at least 64 tiles (32 for the 96- and 128-row tiles of
// 128 columns) and a reduction long enough for splits to fill the GPU (the smallest tile when
// none does); rows are limited by P.  Reduction splits
// then double until the launch has one block per compute unit for the larger tiles, two for the
// smaller ones, keeping at least 8 k tiles per split: more splits cost more in fp32 partial sums
// (written, then read back by a second kernel) than they gain in fill (measured: filling two
// and four per compute unit instead made CIFAR's step 2% slower; half of this, AlexNet's and
// LeNet's 2-5% slower).  kmax (an LDS table limit) can force more splits; the fp32 partial sums
// are capped at 64M elements.
GemmPlan plan_for(int dt, const GemmDims& d)
{
    constexpr long long kTargetTiles = 512, kTargetBlocks = 1024, kMaxPartial = 64ll << 20;
    GemmPlan g{};
    const int fpmax = d.P <= 32 ? 1 : (d.P <= 64 ? 2 : 4);
    static const int cand[5][2] = {{4, 4}, {2, 4}, {2, 2}, {1, 4}, {1, 2}};
    auto tiles = [&](int fp, int fq) {
        return cdiv(d.P, 32 * fp) * cdiv(d.Q, 32 * fq) * (long long)d.Z;
    };
    // k tile: 64, or 32 for short reductions and for the fp32 128 x 128 tile (LDS size)
    auto bk_of = [&](int fp, int fq) {
        return (d.K <= 32 || (dt == DT_F32 && fp == 4 && fq == 4)) ? 32 : 64;
    };
    // bf16: 96-row tiles instead of 128-row ones when P is a multiple of 96 but not of 128
    // (96 or 192 output channels: AlexNet's conv1 and grouped conv4), so that no MFMA rows are
    // padding
    const bool rows96 = dt == DT_BF16 && d.P > 64 && d.P % 96 == 0 && d.P % 128 != 0;
    g.FP = 1;
    g.FQ = 2;
    for (const auto& c0 : cand) {
        int c[2] = {c0[0], c0[1]};
        if (rows96 && c[0] == 4) c[0] = 3;
        if (c[0] > fpmax) continue;
        const long long t = tiles(c[0], c[1]);
        const long long ks = std::min(cdiv(d.K, bk_of(c[0], c[1])) / 8, 32ll);
        // (one 96-row tile stands for two 64-row ones, so it needs half as many tiles; so does
        // the 128 x 128 tile, whose products per LDS byte are twice those of 64 x 64 ones: the
        // CIFAR conv3 weight gradient, 40 tiles over 128 x 577, 74 -> 59 us. Not the 64 x 128
        // tile, which measured slower at 32-63 tiles: CIFAR conv2 112 -> 124 us)
        const long long tmin = c[0] * c[1] >= 12 ? 32 : 64;
        if (t >= kTargetTiles || (t >= tmin && t * ks >= kTargetBlocks)) {
            g.FP = c[0];
            g.FQ = c[1];
            break;
        }
    }
    g.BK = bk_of(g.FP, g.FQ);
    const long long t = tiles(g.FP, g.FQ);
    const long long ktiles = cdiv(d.K, g.BK);
    long long splits = 1;
    const long long slots = 256ll * (g.FP * g.FQ >= 8 ? 1 : 2);
    while (t * splits < slots && ktiles >= 8 * 2 * splits && splits < 256) splits *= 2;
    const long long per_split = (long long)d.P * d.Q * d.Z;
    while (splits > 1 && splits * per_split > kMaxPartial) splits /= 2;
    long long kchunk = cdiv(cdiv(d.K, splits), g.BK) * g.BK;
    if (d.kmax > 0 && kchunk > d.kmax) kchunk = (d.kmax / g.BK) * g.BK;
    if (kchunk < g.BK) kchunk = g.BK;
    g.kchunk = (int)kchunk;
    g.splits = (int)cdiv(d.K, kchunk);
    if (g.splits < 1) g.splits = 1;
    return g;
}

size_t partial_elems(int dt, const GemmDims& d)
{
    const GemmPlan g = plan_for(dt, d);
    if (g.splits <= 1) return 0;
    return (size_t)g.splits * d.Z * (size_t)d.P * d.Q;
}

// GEMM sizes of every operation (P rows, Q columns, reduction, blockIdx.z extent before
// splits, largest reduction chunk with an index table)
GemmDims conv_fwd_dims(int dt, const ConvGeom& g)
{
    const int cg = g.C / g.G, step = cg % vec_elems(dt) == 0 ? vec_elems(dt) : 1;
    return GemmDims{g.OC / g.G, g.N * g.OH * g.OW, g.K * g.K * cg, g.G, kMaxTab * step};
}
GemmDims conv_dgrad_dims(int dt, const ConvGeom& g)
{
    const int og = g.OC / g.G, step = og % vec_elems(dt) == 0 ? vec_elems(dt) : 1;
    return GemmDims{g.C / g.G, g.N * g.H * g.W, g.K * g.K * og, g.G, g.S == 1 ? kMaxTab * step : 0};
}
GemmDims conv_wgrad_dims(int, const ConvGeom& g, int R)
{
    return GemmDims{g.OC / g.G, g.K * g.K * (g.C / g.G) + 1, g.N * g.OH * g.OW, g.G * R, kMaxTab};
}
GemmDims conv_dgrad_col_dims(int, const ConvGeom& g)
{
    return GemmDims{g.K * g.K * (g.C / g.G), g.N * g.OH * g.OW, g.OC / g.G, g.G, 0};
}
size_t conv_dgrad_col_elems(const ConvGeom& g)
{
    return (size_t)g.C * g.K * g.K * (size_t)g.N * g.OH * g.OW;
}
bool conv_dgrad_use_col(const ConvGeom& g)
{
    // taps the implicit GEMM visits per useful multiply-add (stride 1: H*W / (OH*OW)); a strided
    // convolution always takes the col route: its implicit data gradient decodes every tap per
    // element with scalar loads (measured: a 3x3 stride-2 layer of the bottleneck network
    // 875 us implicit)
    const double waste = (double)g.H * g.W / ((double)g.OH * g.OW * g.S * g.S);
    return (waste >= 1.5 || g.S > 1) && conv_dgrad_col_elems(g) * 4 <= (size_t)512 << 20;
}
GemmDims conv_fwd_run_dims(int dt, const ConvGeom& g, const RunGeom& r)
{
    return GemmDims{g.OC, g.N * g.OH * g.OW, g.K * r.RUN, 1, kMaxTab * vec_elems(dt)};
}
GemmDims conv_wgrad_run_dims(int, const ConvGeom& g, const RunGeom& r, int R)
{
    return GemmDims{g.OC, g.K * r.RUN + 1, g.N * g.OH * g.OW, R, kMaxTab};
}
GemmDims fc_fwd_dims(int, int B, int IN, int OUT) { return GemmDims{OUT, B, IN, 1, 0}; }
GemmDims fc_dgrad_dims(int, int B, int IN, int OUT) { return GemmDims{IN, B, OUT, 1, 0}; }
GemmDims fc_wgrad_dims(int, int Nb, int R, int IN, int OUT) { return GemmDims{IN + 1, OUT, Nb, R, 0}; }

}  // namespace mtx
