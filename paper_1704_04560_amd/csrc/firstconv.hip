// Direct kernels for a first convolution with one input channel and a small window (LeNet's
// 1 -> 20 channel 5x5 layer): the implicit GEMM would gather its reduction index k = (u, v)
// with scalar loads and, for the weight gradient, split a 25 x 20 output over long reductions.
// Here the forward computes every output channel of one pixel from its window (fp32 arithmetic,
// the weights as wave-uniform operands), and the weight gradient stages one image in LDS per
// block and reduces over that image's positions in a fixed order; a second kernel adds the
// images of each shard in a fixed order into the shard's gradient row.  No atomics.
#include <algorithm>

#include "device_common.h"
#include "internal.h"
#include "prep.h"

namespace mtx {

// LDS floats of the weight-gradient block: the image and its output gradient as fp32, later
// reused for the sums of the eight thread groups
static size_t first_conv_lds_floats(const ConvGeom& g)
{
    return std::max(((size_t)g.H * g.W + 3) / 4 * 4 + (size_t)g.OH * g.OW * g.OC,
                    (size_t)8 * (g.OC * g.K * g.K + g.OC));
}

// Output rows per forward block: as many whole rows as fit in 256 lanes, evened out over the
// image's rows
// (with a pooling window pk fused in, a multiple of pk, so that no window straddles two blocks;
// 0 when pk rows do not fit)
static int first_conv_rows(const ConvGeom& g, int pk = 1)
{
    int fit = std::max(1, std::min(g.OH, 256 / g.OW));
    fit -= fit % pk;
    if (fit < 1) return 0;
    const int blocks = (g.OH + fit - 1) / fit;
    const int rb = (g.OH + blocks - 1) / blocks;
    return (rb + pk - 1) / pk * pk;
}

// LDS floats of the forward block: its input rows and its output tile
static size_t first_conv_fwd_lds_floats(const ConvGeom& g, int pk = 1)
{
    const int rb = first_conv_rows(g, pk);
    return ((size_t)(rb + g.K - 1) * g.W + 3) / 4 * 4 + (size_t)rb * g.OW * g.OC;
}

bool first_conv_pool_ok(const ConvGeom& g, int pk)
{
    return pk >= 1 && pk * pk <= 255 && g.OH / pk >= 1 && g.OW / pk >= 1 &&
           first_conv_rows(g, pk) >= pk && first_conv_fwd_lds_floats(g, pk) * 4 <= kFirstMaxLds;
}

bool first_conv_direct(const ConvGeom& g, int)
{
    return g.C == 1 && g.G == 1 && g.S == 1 && (g.K == 3 || g.K == 5 || g.K == 7) &&
           g.OC % 4 == 0 && g.OC <= kFirstMaxOC && (g.OC / 4) * g.K <= 32 && g.OW <= 256 &&
           first_conv_lds_floats(g) * 4 <= kFirstMaxLds &&
           first_conv_fwd_lds_floats(g) * 4 <= kFirstMaxLds;
}

// Four consecutive elements as fp32 (16-byte aligned for fp32, 8-byte for bf16), and back
__device__ __forceinline__ float4 load4(const float* p)
{
    return *reinterpret_cast<const float4*>(p);
}
__device__ __forceinline__ float4 load4(const bf16_t* p)
{
    const uint2 v = *reinterpret_cast<const uint2*>(p);
    return make_float4(__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xffff0000u),
                       __uint_as_float(v.y << 16), __uint_as_float(v.y & 0xffff0000u));
}
__device__ __forceinline__ void store4(float* p, float4 v)
{
    *reinterpret_cast<float4*>(p) = v;
}
__device__ __forceinline__ void store4(bf16_t* p, float4 v)
{
    const uint32_t a = f32_to_bf16(v.x) | (uint32_t)f32_to_bf16(v.y) << 16;
    const uint32_t b = f32_to_bf16(v.z) | (uint32_t)f32_to_bf16(v.w) << 16;
    *reinterpret_cast<uint2*>(p) = make_uint2(a, b);
}

// y[n][oh][ow][co] = bias[co] + sum_{u,v} W[co][u][v] * x[n][oh - PD + u][ow - PD + v] (zero
// outside), ReLU.  Block n * tiles + t computes output rows [t * RB, +RB) of image n: the input
// rows it needs are staged in LDS, one thread per output pixel computes all OC channels in fp32
// (the weights, the same for every lane, are wave-uniform operands, rounded to the compute type
// as every other layer's are) into an LDS tile, and the tile, a contiguous range of y, is written
// with 16-byte (fp32) or 8-byte (bf16) stores.
template <typename T, typename TY, int K>
__global__ __launch_bounds__(256) void first_conv_fwd_kernel(const T* __restrict__ x,
                                                             const float* __restrict__ w,
                                                             const float* __restrict__ bias,
                                                             TY* __restrict__ y, int H, int W,
                                                             int OC, int PD, int OH, int OW,
                                                             int RB, int tiles, int relu,
                                                             FirstPoolFwd pool, FirstPrep prep)
{
    if ((int)blockIdx.x >= prep.first) {
        // the weight preparation rides on this launch (nothing of it is read here)
        prep_block<T>(prep.jobs, prep.njobs, prep.w, static_cast<T*>(prep.dst),
                      (int)blockIdx.x - prep.first);
        return;
    }
    constexpr int KK = K * K;
    extern __shared__ __attribute__((aligned(16))) float sm[];
    const int n = blockIdx.x / tiles, oh0 = (blockIdx.x - n * tiles) * RB;  // n < images
    const int rows = min(RB, OH - oh0);
    const int IR = RB + K - 1;
    float* xs = sm;                            // input rows oh0 - PD .. oh0 - PD + IR - 1
    float* ys = sm + (IR * W + 3) / 4 * 4;     // [rows * OW][OC]
    const T* xn = x + (size_t)n * H * W;
    for (int i = threadIdx.x; i < IR * W; i += blockDim.x) {
        const int h = oh0 - PD + i / W;
        xs[i] = (unsigned)h < (unsigned)H ? to_f32<T>(xn[(size_t)h * W + i % W]) : 0.f;
    }
    __syncthreads();
    const int pix = threadIdx.x;
    if (pix < rows * OW) {
        const int r = pix / OW, ow = pix - r * OW;
        float tap[KK];
#pragma unroll
        for (int u = 0; u < K; ++u)
#pragma unroll
            for (int v = 0; v < K; ++v) {
                const int wi = ow - PD + v;
                tap[u * K + v] = (unsigned)wi < (unsigned)W ? xs[(r + u) * W + wi] : 0.f;
            }
        for (int c0 = 0; c0 < OC; c0 += 4) {
            const float* wc = w + c0 * KK;
            float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kk = 0; kk < KK; ++kk)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    acc[j] = fmaf(to_f32<T>(from_f32<T>(wc[j * KK + kk])), tap[kk], acc[j]);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const float a = acc[j] + bias[c0 + j];
                acc[j] = relu ? fmaxf(a, 0.f) : a;
            }
            *reinterpret_cast<float4*>(ys + pix * OC + c0) =
                make_float4(acc[0], acc[1], acc[2], acc[3]);
        }
    }
    __syncthreads();
    TY* yt = y + ((size_t)n * OH + oh0) * OW * OC;
    for (int e = threadIdx.x * 4; e < rows * OW * OC; e += blockDim.x * 4)
        store4(yt + e, *reinterpret_cast<const float4*>(ys + e));
    if (!pool.y) return;
    // The max pooling above (window = stride = PK, NHWC) over the block's rows (RB and oh0 are
    // multiples of PK): per window and 4 channels, the first maximum in row-major window order
    // of the stored (compute-type) outputs, and its window position.
    const int PK = pool.k, PH = OH / PK, PW = OW / PK, CG = OC / 4;
    const int pr0 = oh0 / PK, prows = min(rows / PK, PH - pr0);
    TY* py = static_cast<TY*>(pool.y);
    for (int gi = threadIdx.x; gi < prows * PW * CG; gi += blockDim.x) {
        const int pos = gi / CG, c0 = (gi - pos * CG) * 4;
        const int pr = pos / PW, pw = pos - pr * PW;
        const float* w0 = ys + ((pr * PK) * OW + pw * PK) * OC + c0;
        float bv[4];
        unsigned bi[4] = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int e = 0; e < 4; ++e) bv[e] = to_f32<TY>(from_f32<TY>(w0[e]));
        for (int a = 0; a < PK; ++a)
            for (int b = 0; b < PK; ++b) {
                const float* wp = w0 + (a * OW + b) * OC;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float tv = to_f32<TY>(from_f32<TY>(wp[e]));
                    if (tv > bv[e]) { bv[e] = tv; bi[e] = (unsigned)(a * PK + b); }
                }
            }
        const size_t o = (((size_t)n * PH + pr0 + pr) * PW + pw) * OC + c0;
        store4(py + o, make_float4(bv[0], bv[1], bv[2], bv[3]));
        *reinterpret_cast<unsigned*>(pool.argmax + o) = bi[0] | bi[1] << 8 | bi[2] << 16 | bi[3] << 24;
    }
}

// One block per image n: partial[n][co * KK + kk] = sum over the image's output positions of
// dy[pos][co] * x[tap kk of pos]; partial[n][OC * KK + co] = sum dy[pos][co].  The image and its
// output gradient are staged in LDS with 16-byte (8-byte for bf16) loads, all in flight at once.
// Eight thread groups of 32 take output rows oh = g, g + 8, ...; in a group, thread j owns four
// channels (4 * (j % (OC / 4)) ..) and one window row u = j / (OC / 4): along an output row it
// keeps the K inputs of its window row in registers and shifts them by one position per step, so
// each position costs two LDS reads and 4 x K multiply-adds.  The groups' sums are added in
// ascending group order at the end.
template <typename T, int K>
__global__ __launch_bounds__(256) void first_conv_wgrad_kernel(const T* __restrict__ x,
                                                               const T* __restrict__ dy, int H,
                                                               int W, int OC, int PD, int OH,
                                                               int OW,
                                                               float* __restrict__ partial,
                                                               FirstPool pool)
{
    constexpr int KK = K * K;
    extern __shared__ __attribute__((aligned(16))) float sm[];
    float* xs = sm;                          // [H][W]
    float* ds = sm + (H * W + 3) / 4 * 4;    // [OH * OW][OC]
    const int n = blockIdx.x, NO = OC * KK + OC;
    const int tid = threadIdx.x;
    const T* xn = x + (size_t)n * H * W;
    if (!pool.dy) {
        const T* dn = dy + (size_t)n * OH * OW * OC;
        const int nd = OH * OW * OC;  // a multiple of 4; dn is 8-byte (bf16) / 16-byte aligned
#pragma unroll 4
        for (int e = tid * 4; e < nd; e += 1024)
            *reinterpret_cast<float4*>(ds + e) = load4(dn + e);
    } else {
        // The output gradient comes from the max pooling above (window = stride = PK, NHWC):
        // every position of a window gets the window's gradient if it holds the window's
        // maximum, else 0 (and the window passes nothing where a ReLU on this layer made the
        // pooled output non-positive); positions no window covers get 0.
        const int PK = pool.k, PH = OH / PK, PW = OW / PK, CG = OC / 4;
        const int ng = PH * PW * CG;
        const T* gp = static_cast<const T*>(pool.dy) + (size_t)n * PH * PW * OC;
        const uint8_t* ap = pool.argmax + (size_t)n * PH * PW * OC;
        const T* yp = static_cast<const T*>(pool.gate);
        if (yp) yp += (size_t)n * PH * PW * OC;
        constexpr int kU = 4;  // window groups per thread and batch: all loads before the stores
        for (int b0 = 0; b0 < ng; b0 += 256 * kU) {
            float4 gv[kU];
            unsigned am[kU];
#pragma unroll
            for (int u = 0; u < kU; ++u) {
                const int gi = b0 + 256 * u + tid;
                gv[u] = make_float4(0.f, 0.f, 0.f, 0.f);
                am[u] = 0xffffffffu;
                if (gi < ng) {
                    const int o = (gi / CG) * OC + (gi % CG) * 4;
                    gv[u] = load4(gp + o);
                    am[u] = *reinterpret_cast<const unsigned*>(ap + o);
                    if (yp) {
                        const float4 y = load4(yp + o);
                        if (!(y.x > 0.f)) gv[u].x = 0.f;
                        if (!(y.y > 0.f)) gv[u].y = 0.f;
                        if (!(y.z > 0.f)) gv[u].z = 0.f;
                        if (!(y.w > 0.f)) gv[u].w = 0.f;
                    }
                }
            }
#pragma unroll
            for (int u = 0; u < kU; ++u) {
                const int gi = b0 + 256 * u + tid;
                if (gi >= ng) continue;
                const int pos = gi / CG, c0 = (gi % CG) * 4;
                const int ph = pos / PW, pw = pos - ph * PW;
                for (int a = 0; a < PK; ++a)
                    for (int b = 0; b < PK; ++b) {
                        const unsigned wpos = (unsigned)(a * PK + b);
                        const float4 v = make_float4(
                            (am[u] & 0xffu) == wpos ? gv[u].x : 0.f,
                            ((am[u] >> 8) & 0xffu) == wpos ? gv[u].y : 0.f,
                            ((am[u] >> 16) & 0xffu) == wpos ? gv[u].z : 0.f,
                            (am[u] >> 24) == wpos ? gv[u].w : 0.f);
                        const int oh = ph * PK + a, ow = pw * PK + b;
                        *reinterpret_cast<float4*>(ds + (oh * OW + ow) * OC + c0) = v;
                    }
            }
        }
        if (OH != PH * PK || OW != PW * PK) {
            for (int e = tid * 4; e < OH * OW * OC; e += 1024) {
                const int pos = e / OC, oh = pos / OW, ow = pos - oh * OW;
                if (oh >= PH * PK || ow >= PW * PK)
                    *reinterpret_cast<float4*>(ds + e) = make_float4(0.f, 0.f, 0.f, 0.f);
            }
        }
    }
    for (int i = tid; i < H * W; i += 256) xs[i] = to_f32<T>(xn[i]);
    __syncthreads();
    const int grp = tid >> 5, j = tid & 31;
    const int ncg = OC / 4, active = ncg * K;
    float acc[4][K], bacc[4];
#pragma unroll
    for (int a = 0; a < 4; ++a) {
        bacc[a] = 0.f;
#pragma unroll
        for (int v = 0; v < K; ++v) acc[a][v] = 0.f;
    }
    const int cg = j % ncg, u = j / ncg, c0 = 4 * cg;
    if (j < active) {
        for (int oh = grp; oh < OH; oh += 8) {
            const int h = oh - PD + u;
            const bool hok = (unsigned)h < (unsigned)H;
            const float* xr = xs + (hok ? h : 0) * W;
            // win[v] = x[h][ow - PD + v] for the current ow
            float win[K];
#pragma unroll
            for (int v = 0; v < K - 1; ++v) {
                const int wi = v - PD;
                win[v + 1] = (hok && (unsigned)wi < (unsigned)W) ? xr[wi] : 0.f;
            }
            const float* drow = ds + oh * OW * OC + c0;
#pragma unroll 4
            for (int ow = 0; ow < OW; ++ow) {
#pragma unroll
                for (int v = 0; v < K - 1; ++v) win[v] = win[v + 1];
                const int wi = ow - PD + K - 1;
                win[K - 1] = (hok && (unsigned)wi < (unsigned)W) ? xr[wi] : 0.f;
                const float4 g = *reinterpret_cast<const float4*>(drow + ow * OC);
                const float gv[4] = {g.x, g.y, g.z, g.w};
#pragma unroll
                for (int a = 0; a < 4; ++a) {
#pragma unroll
                    for (int v = 0; v < K; ++v) acc[a][v] = fmaf(gv[a], win[v], acc[a][v]);
                    bacc[a] += gv[a];
                }
            }
        }
    }
    __syncthreads();  // the staged tensors are no longer read; reuse the LDS for the group sums
    float* red = sm;  // [8][NO]
    if (j < active) {
#pragma unroll
        for (int a = 0; a < 4; ++a) {
#pragma unroll
            for (int v = 0; v < K; ++v) red[grp * NO + (c0 + a) * KK + u * K + v] = acc[a][v];
            if (u == 0) red[grp * NO + OC * KK + c0 + a] = bacc[a];
        }
    }
    __syncthreads();
    for (int o = tid; o < NO; o += 256) {
        float s = 0.f;
        for (int q = 0; q < 8; ++q) s += red[q * NO + o];
        partial[(size_t)n * NO + o] = s;
    }
}

// grads[r * ld + w_off + o] (o < OC*KK) and grads[r * ld + b_off + co]: the sum over the shard's
// Nb images.  Block (r, chunk) owns 64 consecutive outputs; its four waves add the images
// q, q + 4, ... (ascending) and the four sums are added in ascending q.
__global__ __launch_bounds__(256) void first_conv_wgrad_reduce_kernel(
    const float* __restrict__ partial, int Nb, int NO, int OCKK, float* __restrict__ grads,
    long long ld, long long w_off, long long b_off)
{
    __shared__ float red[4][64];
    const int r = blockIdx.y, q = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int o = blockIdx.x * 64 + lane;
    float s = 0.f;
    if (o < NO) {
        const float* p = partial + (size_t)r * Nb * NO + o;
#pragma unroll 4
        for (int i = q; i < Nb; i += 4) s += p[(size_t)i * NO];
    }
    red[q][lane] = s;
    __syncthreads();
    if (q == 0 && o < NO) {
        const float t = ((red[0][lane] + red[1][lane]) + red[2][lane]) + red[3][lane];
        const long long dst = o < OCKK ? w_off + o : b_off + (o - OCKK);
        grads[(long long)r * ld + dst] = t;
    }
}

hipError_t first_conv_fwd(Dt dt, const ConvGeom& g, const void* x, const float* w,
                          const float* bias, void* y, bool y_f32, bool relu, hipStream_t s,
                          const FirstPoolFwd& pool, const FirstPrep& prep)
{
    if (!first_conv_direct(g, dt)) return hipErrorInvalidValue;
    const int pk = pool.y ? pool.k : 1;
    if (pool.y && (!first_conv_pool_ok(g, pk) || (y_f32 && dt != DT_F32)))
        return hipErrorInvalidValue;  // the pooled output has the conv output's type
    const int rb = first_conv_rows(g, pk);
    const int tiles = (g.OH + rb - 1) / rb;
    // blocks [0, tiles * N): the convolution; then the preparation blocks (256 threads each)
    FirstPrep pr = prep;
    pr.first = tiles * g.N;
    if (pr.blocks < 0 || (pr.blocks > 0 && (!pr.jobs || pr.njobs < 1 || !pr.dst || !pr.w)))
        return hipErrorInvalidValue;
    const dim3 grid(tiles * g.N + pr.blocks);
    const int threads = pr.blocks > 0 ? 256 : (rb * g.OW + 63) / 64 * 64;
    const size_t shm = first_conv_fwd_lds_floats(g, pk) * 4;
    auto go = [&](auto kern, const auto* xt, auto* yt) {
        hipLaunchKernelGGL(kern, grid, dim3(threads), shm, s, xt, w, bias, yt, g.H, g.W, g.OC,
                           g.PD, g.OH, g.OW, rb, tiles, relu ? 1 : 0, pool, pr);
    };
    float* yf = static_cast<float*>(y);
    if (dt == DT_F32) {
        const float* xf = static_cast<const float*>(x);
        if (g.K == 3) go(first_conv_fwd_kernel<float, float, 3>, xf, yf);
        else if (g.K == 5) go(first_conv_fwd_kernel<float, float, 5>, xf, yf);
        else go(first_conv_fwd_kernel<float, float, 7>, xf, yf);
    } else if (y_f32) {
        const bf16_t* xb = static_cast<const bf16_t*>(x);
        if (g.K == 3) go(first_conv_fwd_kernel<bf16_t, float, 3>, xb, yf);
        else if (g.K == 5) go(first_conv_fwd_kernel<bf16_t, float, 5>, xb, yf);
        else go(first_conv_fwd_kernel<bf16_t, float, 7>, xb, yf);
    } else {
        const bf16_t* xb = static_cast<const bf16_t*>(x);
        bf16_t* yb = static_cast<bf16_t*>(y);
        if (g.K == 3) go(first_conv_fwd_kernel<bf16_t, bf16_t, 3>, xb, yb);
        else if (g.K == 5) go(first_conv_fwd_kernel<bf16_t, bf16_t, 5>, xb, yb);
        else go(first_conv_fwd_kernel<bf16_t, bf16_t, 7>, xb, yb);
    }
    return hipGetLastError();
}

size_t first_conv_partial_floats(const ConvGeom& g, int R)
{
    return (size_t)R * g.N * (g.OC * g.K * g.K + g.OC);
}

hipError_t first_conv_wgrad(Dt dt, const ConvGeom& g, int R, const void* x, const void* dy,
                            float* partial, float* grads, long long ld, long long w_off,
                            long long b_off, hipStream_t s, const FirstPool& pool)
{
    if (pool.dy && (pool.k < 1 || g.OH / pool.k < 1 || g.OW / pool.k < 1 ||
                    pool.k * pool.k > 255))
        return hipErrorInvalidValue;
    if (!first_conv_direct(g, dt)) return hipErrorInvalidValue;
    const int NO = g.OC * g.K * g.K + g.OC;
    const size_t shm = first_conv_lds_floats(g) * 4;
    const dim3 grid(R * g.N);  // g.N images per shard
    auto go = [&](auto kern, const auto* xt, const auto* dt_) {
        hipLaunchKernelGGL(kern, grid, dim3(256), shm, s, xt, dt_, g.H, g.W, g.OC, g.PD, g.OH,
                           g.OW, partial, pool);
    };
    if (dt == DT_F32) {
        const float* xf = static_cast<const float*>(x);
        const float* df = static_cast<const float*>(dy);
        if (g.K == 3) go(first_conv_wgrad_kernel<float, 3>, xf, df);
        else if (g.K == 5) go(first_conv_wgrad_kernel<float, 5>, xf, df);
        else go(first_conv_wgrad_kernel<float, 7>, xf, df);
    } else {
        const bf16_t* xb = static_cast<const bf16_t*>(x);
        const bf16_t* db = static_cast<const bf16_t*>(dy);
        if (g.K == 3) go(first_conv_wgrad_kernel<bf16_t, 3>, xb, db);
        else if (g.K == 5) go(first_conv_wgrad_kernel<bf16_t, 5>, xb, db);
        else go(first_conv_wgrad_kernel<bf16_t, 7>, xb, db);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    timing_split(s, "reduce");
    hipLaunchKernelGGL(first_conv_wgrad_reduce_kernel, dim3((NO + 63) / 64, R), dim3(256), 0, s,
                       partial, g.N, NO, g.OC * g.K * g.K, grads, ld, w_off, b_off);
    return hipGetLastError();
}

}  // namespace mtx
