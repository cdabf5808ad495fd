// Data gradient of a small-image fp32 convolution in one kernel (LeNet's second layer: 20 -> 50
// channels, 5x5, 12x12 -> 8x8).  The col route (col = Wc . dy as a matrix product into an fp32
// buffer, then col2im) writes and re-reads C*K*K values per output position through HBM; here a
// block owns one image and a range of input channels, computes that image's col tile on the
// matrix cores into LDS and folds it into dx from there.  The arithmetic is the col route's:
// every col value is one sum over the output channels, and dx adds the col values of the taps
// (u, v) in ascending order; only the memory traffic differs.
#include <algorithm>

#include "device_common.h"
#include "internal.h"

namespace mtx {

namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kDxMaxPos = 64;    // output positions per image: at most 4 column tiles of 16
constexpr int kDxMaxRows = 256;  // (tap, channel) rows per block: at most 16 row tiles of 16

// A block's matrix product is always 16 x 4 tiles of 16 x 16: rows r = cl * K * K + (u * K + v)
// for the block's channels cl (at most 256 rows), columns the output positions (at most 64);
// rows and columns beyond the problem are zero, so the product loop has no conditions.
constexpr int kDxRS = kDxMaxRows + 16;  // LDS row stride of the k-major weight operand

struct DxShape {
    int cb;      // input channels per block
    int chunks;  // blocks per image
    int ps;      // LDS row stride of the col tile (odd)
    size_t lds;  // LDS floats
};

DxShape dx_shape(const ConvGeom& g)
{
    DxShape s{};
    const int cbmax = kDxMaxRows / (g.K * g.K);
    s.chunks = (g.C + cbmax - 1) / cbmax;
    s.cb = (g.C + s.chunks - 1) / s.chunks;
    const int ks = (g.OC + 3) / 4;
    s.ps = (g.OH * g.OW) | 1;
    const size_t ab = (size_t)4 * ks * kDxRS + (size_t)kDxMaxPos * g.OC + 4;
    const size_t col = (size_t)kDxMaxRows * s.ps;
    s.lds = std::max(ab, col);
    return s;
}

// Block n * chunks + j: input channels [c0, c0 + cbc), c0 = j * CB, of image n.
//   col[r][p] = sum_co W[co][c0 + cl][u][v] * dy[n][p][co],   r = cl * K * K + u * K + v
//   dx[n][h][w][c0 + cl] = mask * sum_{u, v ascending} col[r][oh * OW + ow]
//                          with oh = h + PD - u, ow = w + PD - v inside the output.
// W is the fp32 weight tensor [OC][C][K][K]: for one output channel the block's rows are one
// contiguous run, staged k-major (As[co][r]); the image's dy is one contiguous run, staged as it
// is (Bs[p * OC + co]; the reads past a row's end meet zero rows of As, and the positions past
// the image are zero).  Both are copied with 16-byte loads, every load of a thread issued before
// any LDS write, so that the block waits for memory once.
// The product runs as v_mfma_f32_16x16x4_f32: wave wv owns row tiles wv, wv + 4, wv + 8,
// wv + 12 and the four column tiles; lane l supplies row l % 16 and k = 4 * step + l / 16 of
// both operands, and holds rows 4 * (l / 16) + v, column l % 16 of the result.
template <int K>
__global__ __launch_bounds__(256) void dgrad_fused_kernel(const float* __restrict__ dy,
                                                          const float* __restrict__ w,
                                                          float* __restrict__ dx,
                                                          const void* __restrict__ mask,
                                                          int mask_f32, int C, int H, int W,
                                                          int OC, int OH, int OW, int PD, int CB,
                                                          int chunks, int PS)
{
    constexpr int KK = K * K;
    constexpr int CBMAX = kDxMaxRows / KK;
    extern __shared__ __attribute__((aligned(16))) float sm[];
    const int n = blockIdx.x / chunks, j = blockIdx.x - n * chunks;
    const int c0 = j * CB, cbc = min(CB, C - c0);
    const int Mb = cbc * KK, P = OH * OW;
    const int KS = (OC + 3) / 4;
    float* As = sm;                  // [4 * KS][kDxRS]
    float* Bs = sm + 4 * KS * kDxRS; // [kDxMaxPos * OC + 4]
    const int tid = threadIdx.x;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
    {
        // A: item i = (k = i / 64, four rows 4 * (i % 64) ..); B: four floats 4 * e ..
        constexpr int AI = 64 * 64 / 256, BI = (kDxMaxPos * 64 + 4 + 1023) / 1024;
        float4 va[AI], vb[BI];
        const float* wr = w + (size_t)c0 * KK;
        const size_t wsk = (size_t)C * KK;
#pragma unroll
        for (int it = 0; it < AI; ++it) {
            const int i = tid + 256 * it, k = i >> 6, r = 4 * (i & 63);
            va[it] = make_float4(0.f, 0.f, 0.f, 0.f);
            if (k < OC) {
                const float* src = wr + k * wsk + r;
                if (r + 3 < Mb) {
                    __builtin_memcpy(&va[it], src, 16);
                } else {
                    if (r < Mb) va[it].x = src[0];
                    if (r + 1 < Mb) va[it].y = src[1];
                    if (r + 2 < Mb) va[it].z = src[2];
                }
            }
        }
        const float* dn = dy + (size_t)n * P * OC;
        const int nb = P * OC, nz = kDxMaxPos * OC + 4;
#pragma unroll
        for (int it = 0; it < BI; ++it) {
            const int e = 4 * (tid + 256 * it);
            vb[it] = make_float4(0.f, 0.f, 0.f, 0.f);
            if (e + 3 < nb) {
                __builtin_memcpy(&vb[it], dn + e, 16);
            } else {
                if (e < nb) vb[it].x = dn[e];
                if (e + 1 < nb) vb[it].y = dn[e + 1];
                if (e + 2 < nb) vb[it].z = dn[e + 2];
            }
        }
#pragma unroll
        for (int it = 0; it < AI; ++it) {
            const int i = tid + 256 * it, k = i >> 6, r = 4 * (i & 63);
            if (k < 4 * KS) *reinterpret_cast<float4*>(As + k * kDxRS + r) = va[it];
        }
#pragma unroll
        for (int it = 0; it < BI; ++it) {
            const int e = 4 * (tid + 256 * it);
            if (e < nz) *reinterpret_cast<float4*>(Bs + e) = vb[it];
        }
    }
    __syncthreads();

    const int lane = tid & 63, lr = lane & 15, lg = lane >> 4;
    f32x4 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int t = 0; t < 4; ++t) acc[i][t] = f32x4{0.f, 0.f, 0.f, 0.f};
    const float* ap = As + lg * kDxRS + wv * 16 + lr;
    const float* bp = Bs + lr * OC + lg;
    float a[4], b[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) b[t] = bp[t * 16 * OC];
#pragma unroll
    for (int i = 0; i < 4; ++i) a[i] = ap[i * 64];
    for (int ks = 0; ks < KS; ++ks) {
        // the next step's operands (the first step's again after the last) while these run
        const int kn = ks + 1 < KS ? (ks + 1) * 4 : 0;
        float an[4], bn[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) bn[t] = bp[t * 16 * OC + kn];
#pragma unroll
        for (int i = 0; i < 4; ++i) an[i] = ap[i * 64 + kn * kDxRS];
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                acc[i][t] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], b[t], acc[i][t], 0, 0, 0);
#pragma unroll
        for (int q = 0; q < 4; ++q) { a[q] = an[q]; b[q] = bn[q]; }
    }
    __syncthreads();  // the operands are consumed; the col tile takes their place
    float* cs = sm;   // [kDxMaxRows][PS]
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const int p = t * 16 + lr;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int r = (wv + 4 * i) * 16 + 4 * lg + v;
                if (p < P) cs[r * PS + p] = acc[i][t][v];
            }
        }
    }
    __syncthreads();
    // col2im: one thread per input position, all channels of the block; the taps that land
    // inside the output form a rectangle of (u, v), visited in ascending order
    const int HW = H * W;
    for (int hw = tid; hw < HW; hw += 256) {
        const int h = hw / W, wq = hw - h * W;
        float accs[CBMAX];
#pragma unroll
        for (int cl = 0; cl < CBMAX; ++cl) accs[cl] = 0.f;
        const int u_lo = max(0, h + PD - OH + 1), u_hi = min(K - 1, h + PD);
        const int v_lo = max(0, wq + PD - OW + 1), v_hi = min(K - 1, wq + PD);
        for (int u = u_lo; u <= u_hi; ++u)
            for (int v = v_lo; v <= v_hi; ++v) {
                const float* c = cs + (u * K + v) * PS + (h + PD - u) * OW + (wq + PD - v);
#pragma unroll
                for (int cl = 0; cl < CBMAX; ++cl) accs[cl] += c[cl * KK * PS];
            }
        const size_t o = ((size_t)n * HW + hw) * C + c0;
#pragma unroll
        for (int cl = 0; cl < CBMAX; ++cl) {
            if (cl >= cbc) break;
            float r = accs[cl];
            if (mask) {
                const float m = mask_f32 ? static_cast<const float*>(mask)[o + cl]
                                         : bf16_to_f32(static_cast<const bf16_t*>(mask)[o + cl]);
                if (!(m > 0.f)) r = 0.f;
            }
            dx[o + cl] = r;
        }
    }
}

}  // namespace

bool conv_dgrad_fused_ok(const ConvGeom& g, int dt)
{
    if (dt != DT_F32 || g.G != 1 || g.S != 1 || !(g.K == 3 || g.K == 5)) return false;
    if (g.OH * g.OW > kDxMaxPos || g.K * g.K > kDxMaxRows || g.OC > 60) return false;
    return dx_shape(g).lds * 4 <= kDxMaxLds;
}

hipError_t conv_dgrad_fused(const ConvGeom& g, const float* dy, const float* w, float* dx,
                            const void* mask, bool mask_f32, hipStream_t s)
{
    if (!conv_dgrad_fused_ok(g, DT_F32)) return hipErrorInvalidValue;
    const DxShape d = dx_shape(g);
    const dim3 grid((unsigned)g.N * d.chunks);
    auto go = [&](auto kern) {
        hipLaunchKernelGGL(kern, grid, dim3(256), d.lds * 4, s, dy, w, dx, mask,
                           mask_f32 ? 1 : 0, g.C, g.H, g.W, g.OC, g.OH, g.OW, g.PD, d.cb,
                           d.chunks, d.ps);
    };
    if (g.K == 3) go(dgrad_fused_kernel<3>);
    else go(dgrad_fused_kernel<5>);
    return hipGetLastError();
}

}  // namespace mtx
