// Batch normalisation with per-shard statistics and the residual addition (the building blocks
// of the ResNet-50 network in Table II), over NHWC tensors [R*Nb][H*W][C] of all R shards.
//
// Batch normalisation normalises channel c of shard r by the mean and the biased variance of
// its M = Nb*H*W values: y = gamma (x - mean) / sqrt(var + eps) + beta.  The per-shard sums are
// reductions over rows: a block takes a contiguous range of one shard's rows (one of S splits)
// and every channel, adds in fp32 over short runs and in double across runs, and writes one
// partial per (shard, split, channel); a finalize kernel adds the S partials in ascending order.
// No atomics: results are the same on every run.  Per-channel values are kept as planes
// [R][plane][C] so that a thread reads those of its channels as whole vectors.  Channel counts
// that are a multiple of the 16-byte vector width V (and at most 256 V) use 16-byte loads and
// stores; the others take one element per thread.
#include "device_common.h"
#include "internal.h"

namespace mtx {

// planes of the forward statistics [R][kStatPlanes][C]
enum { ST_MEAN = 0, ST_INV = 1, ST_SCALE = 2, ST_SHIFT = 3, kStatPlanes = 4 };
// planes of the backward coefficients [R][3][C]: dx = k1 (dy - k2 - xhat k3)
enum { CO_K1 = 0, CO_K2 = 1, CO_K3 = 2, kCoefPlanes = 3 };

typedef unsigned u32x4v __attribute__((ext_vector_type(4)));
constexpr int kUnroll = 4;  // rows a thread loads before adding them

template <typename T, int V>
__device__ __forceinline__ void load_vec(const T* p, float (&v)[V])
{
    const u32x4v raw = *reinterpret_cast<const u32x4v*>(p);
    const T* e = reinterpret_cast<const T*>(&raw);
#pragma unroll
    for (int i = 0; i < V; ++i) v[i] = to_f32<T>(e[i]);
}

template <typename T, int V>
__device__ __forceinline__ void store_vec(T* p, const float (&v)[V])
{
    u32x4v raw;
    T* e = reinterpret_cast<T*>(&raw);
#pragma unroll
    for (int i = 0; i < V; ++i) e[i] = from_f32<T>(v[i]);
    *reinterpret_cast<u32x4v*>(p) = raw;
}

// V consecutive floats of a plane (16-byte aligned when V is 4 or 8 and c0 a multiple of V)
template <int V>
__device__ __forceinline__ void load_plane(const float* p, float (&v)[V])
{
#pragma unroll
    for (int i = 0; i < V; i += 4) {
        const float4 q = *reinterpret_cast<const float4*>(p + i);
        v[i] = q.x;
        v[i + 1] = q.y;
        v[i + 2] = q.z;
        v[i + 3] = q.w;
    }
}

// A ReLU mask read from the stored output of a layer (fp32 or the compute type).
template <typename T>
__device__ __forceinline__ bool mask_pass(const void* m, int m_f32, size_t t)
{
    if (!m) return true;
    const float v = m_f32 ? static_cast<const float*>(m)[t] : to_f32<T>(static_cast<const T*>(m)[t]);
    return v > 0.f;
}

// Row sums of shard r = blockIdx.y over split s = blockIdx.x, for W channels per thread (W = V
// with 16-byte loads, else 1): thread tid takes channel group cg = tid % G (G = ceil(C / W)) and
// row lane rl = tid / G.
//   forward:  (sum x, sum x^2)
//   backward: (sum dy, sum dy * xhat), xhat = (x - mean) * inv
template <typename T, bool BWD, int W>
__global__ __launch_bounds__(256) void bn_partial_kernel(const T* __restrict__ x,
                                                         const T* __restrict__ dy,
                                                         const float* __restrict__ stats,
                                                         int Nb, int HW, int C, int S,
                                                         double* __restrict__ part)
{
    extern __shared__ double red[];  // [2][256][W]
    const int G = (C + W - 1) / W, lanes = 256 / G;
    const int tid = threadIdx.x, cg = tid % G, rl = tid / G;
    const int s = blockIdx.x, r = blockIdx.y;
    const int c0 = cg * W;
    const long long M = (long long)Nb * HW;
    const long long per = (M + S - 1) / S;
    const long long r0 = (long long)s * per, r1 = min(M, r0 + per);
    double da[W], db[W];
#pragma unroll
    for (int k = 0; k < W; ++k) da[k] = db[k] = 0.0;
    if (rl < lanes && c0 < C) {
        float mean[W], inv[W];
#pragma unroll
        for (int k = 0; k < W; ++k) mean[k] = inv[k] = 0.f;
        if (BWD) {
            const float* st = stats + (size_t)r * kStatPlanes * C + c0;
            if constexpr (W > 1) {
                load_plane<W>(st + ST_MEAN * C, mean);
                load_plane<W>(st + ST_INV * C, inv);
            } else {
                mean[0] = st[ST_MEAN * C];
                inv[0] = st[ST_INV * C];
            }
        }
        const T* xb = x + (long long)r * M * C + c0;
        const T* gb = BWD ? dy + (long long)r * M * C + c0 : nullptr;
        // Raw rows (W elements each), loaded one batch of kUnroll rows ahead: the loads of the
        // next batch are in flight while this one is added (with one batch at a time, each
        // thread waited a full memory round trip per batch).  Rows past the range read as zeros.
        typedef std::conditional_t<(W > 1), u32x4v, T> Raw;
        auto load_batch = [&](long long i0, Raw (&rx)[kUnroll], Raw (&rg)[kUnroll]) {
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                const long long i = i0 + (long long)u * lanes;
                rx[u] = Raw{};
                rg[u] = Raw{};
                if (i < r1) {
                    rx[u] = *reinterpret_cast<const Raw*>(xb + i * C);
                    if (BWD) rg[u] = *reinterpret_cast<const Raw*>(gb + i * C);
                }
            }
        };
        auto unpack = [&](const Raw& raw, float (&v)[W]) {
            const T* e = reinterpret_cast<const T*>(&raw);
#pragma unroll
            for (int k = 0; k < W; ++k) v[k] = to_f32<T>(e[k]);
        };
        const long long step = (long long)kUnroll * lanes;
        Raw cx[kUnroll], cg[kUnroll];
        long long i0 = r0 + rl;
        if (i0 < r1) load_batch(i0, cx, cg);
        for (; i0 < r1; i0 += step) {
            Raw nx[kUnroll], ng[kUnroll];
            if (i0 + step < r1) load_batch(i0 + step, nx, ng);
            float xv[kUnroll][W], gv[kUnroll][W];
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                unpack(cx[u], xv[u]);
                if (BWD) unpack(cg[u], gv[u]);
                else
#pragma unroll
                    for (int k = 0; k < W; ++k) gv[u][k] = 0.f;
            }
            float fa[W], fb[W];
#pragma unroll
            for (int k = 0; k < W; ++k) fa[k] = fb[k] = 0.f;
#pragma unroll
            for (int u = 0; u < kUnroll; ++u)
#pragma unroll
                for (int k = 0; k < W; ++k) {
                    if (!BWD) {
                        fa[k] += xv[u][k];
                        fb[k] = fmaf(xv[u][k], xv[u][k], fb[k]);
                    } else {
                        fa[k] += gv[u][k];
                        fb[k] = fmaf(gv[u][k], (xv[u][k] - mean[k]) * inv[k], fb[k]);
                    }
                }
#pragma unroll
            for (int k = 0; k < W; ++k) {
                da[k] += (double)fa[k];
                db[k] += (double)fb[k];
            }
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                cx[u] = nx[u];
                cg[u] = ng[u];
            }
        }
    }
#pragma unroll
    for (int k = 0; k < W; ++k) {
        red[(size_t)tid * W + k] = da[k];
        red[(size_t)(256 + tid) * W + k] = db[k];
    }
    __syncthreads();
    // one thread per channel adds the row lanes of its group in ascending order
    for (int c = tid; c < C; c += 256) {
        const int g = c / W, k = c - g * W;
        double a = 0.0, b = 0.0;
        for (int l = 0; l < lanes; ++l) {
            a += red[(size_t)(l * G + g) * W + k];
            b += red[(size_t)(256 + l * G + g) * W + k];
        }
        double* p = part + (((long long)r * S + s) * C + c) * 2;
        p[0] = a;
        p[1] = b;
    }
}

// Per (shard, channel) from the S partials: a block covers 64 channels of one shard, lane q of
// four adds splits q, q + 4, ... and the four are added in ascending q.  Then
//   forward:  mean, inv = 1 / sqrt(var + eps) (var = E[x^2] - mean^2 in double),
//             scale = gamma * inv, shift = beta;
//   backward: the shard's gamma and beta gradients (rows of grads) and the coefficients of
//             dx = k1 (dy - k2 - xhat k3): k1 = gamma * inv, k2 = sum dy / M, k3 = sum(dy xhat) / M.
template <bool BWD>
__global__ __launch_bounds__(256) void bn_finalize_kernel(
    const double* __restrict__ part, int C, int S, long long M, double eps,
    const float* __restrict__ gamma, const float* __restrict__ beta, float* __restrict__ stats,
    float* __restrict__ grads, long long ld, long long w_off, long long b_off,
    float* __restrict__ coef)
{
    const int lane = threadIdx.x & 63, q = threadIdx.x >> 6;
    const int c = blockIdx.x * 64 + lane, r = blockIdx.y;
    double a = 0.0, b = 0.0;
    if (c < C) {
#pragma unroll 8
        for (int s = q; s < S; s += 4) {
            const double* p = part + (((long long)r * S + s) * C + c) * 2;
            a += p[0];
            b += p[1];
        }
    }
    __shared__ double sa[4][64], sb[4][64];
    sa[q][lane] = a;
    sb[q][lane] = b;
    __syncthreads();
    if (q != 0 || c >= C) return;
    a = ((sa[0][lane] + sa[1][lane]) + sa[2][lane]) + sa[3][lane];
    b = ((sb[0][lane] + sb[1][lane]) + sb[2][lane]) + sb[3][lane];
    float* st = stats + (size_t)r * kStatPlanes * C + c;
    if (!BWD) {
        const double mean = a / (double)M;
        const double var = fmax(b / (double)M - mean * mean, 0.0);
        const float inv = (float)(1.0 / sqrt(var + eps));
        st[ST_MEAN * C] = (float)mean;
        st[ST_INV * C] = inv;
        st[ST_SCALE * C] = gamma[c] * inv;
        st[ST_SHIFT * C] = beta[c];
    } else {
        grads[(long long)r * ld + w_off + c] = (float)b;
        grads[(long long)r * ld + b_off + c] = (float)a;
        float* co = coef + (size_t)r * kCoefPlanes * C + c;
        co[CO_K1 * C] = st[ST_SCALE * C];
        co[CO_K2 * C] = (float)(a / (double)M);
        co[CO_K3 * C] = (float)(b / (double)M);
    }
}

// y = (x - mean) * scale + shift, ReLU, stored in the compute type; W consecutive channels per
// thread (the element index t counts groups of W).
template <typename T, int W>
// (skip != null: the residual addition that follows, z = y + skip with its own ReLU flag, in the
// same pass: y as stored, plus skip, rounded once -- the arithmetic of add_fwd_kernel)
__global__ __launch_bounds__(256) void bn_apply_kernel(const T* __restrict__ x, T* __restrict__ y,
                                                       const float* __restrict__ stats,
                                                       unsigned rows_per_shard, int C,
                                                       unsigned n, int relu,
                                                       const T* __restrict__ skip,
                                                       T* __restrict__ z, int relu2)
{
    const unsigned t = blockIdx.x * 256 + threadIdx.x;
    if (t >= n) return;
    const size_t e = (size_t)t * W;
    const unsigned row = (unsigned)(e / (unsigned)C), c0 = (unsigned)(e - (size_t)row * C);
    const float* st = stats + (size_t)(row / rows_per_shard) * kStatPlanes * C + c0;
    float v[W], mean[W], sc[W], sh[W];
    if constexpr (W > 1) {
        load_vec<T, W>(x + e, v);
        load_plane<W>(st + ST_MEAN * C, mean);
        load_plane<W>(st + ST_SCALE * C, sc);
        load_plane<W>(st + ST_SHIFT * C, sh);
    } else {
        v[0] = to_f32<T>(x[e]);
        mean[0] = st[ST_MEAN * C];
        sc[0] = st[ST_SCALE * C];
        sh[0] = st[ST_SHIFT * C];
    }
#pragma unroll
    for (int k = 0; k < W; ++k) {
        v[k] = fmaf(v[k] - mean[k], sc[k], sh[k]);
        if (relu) v[k] = fmaxf(v[k], 0.f);
    }
    if constexpr (W > 1) store_vec<T, W>(y + e, v);
    else y[e] = from_f32<T>(v[0]);
    if (skip) {
        float b[W];
        if constexpr (W > 1) load_vec<T, W>(skip + e, b);
        else b[0] = to_f32<T>(skip[e]);
#pragma unroll
        for (int k = 0; k < W; ++k) {
            v[k] = to_f32<T>(from_f32<T>(v[k])) + b[k];
            if (relu2) v[k] = fmaxf(v[k], 0.f);
        }
        if constexpr (W > 1) store_vec<T, W>(z + e, v);
        else z[e] = from_f32<T>(v[0]);
    }
}

template <typename T, int W>
__global__ __launch_bounds__(256) void bn_bwd_apply_kernel(
    const T* __restrict__ x, const T* __restrict__ dy, const float* __restrict__ stats,
    const float* __restrict__ coef, const void* mask, int mask_f32, T* __restrict__ dx,
    unsigned rows_per_shard, int C, unsigned n)
{
    const unsigned t = blockIdx.x * 256 + threadIdx.x;
    if (t >= n) return;
    const size_t e = (size_t)t * W;
    const unsigned row = (unsigned)(e / (unsigned)C), c0 = (unsigned)(e - (size_t)row * C);
    const size_t r = row / rows_per_shard;
    const float* st = stats + r * kStatPlanes * C + c0;
    const float* co = coef + r * kCoefPlanes * C + c0;
    float xv[W], g[W], mean[W], inv[W], k1[W], k2[W], k3[W];
    if constexpr (W > 1) {
        load_vec<T, W>(x + e, xv);
        load_vec<T, W>(dy + e, g);
        load_plane<W>(st + ST_MEAN * C, mean);
        load_plane<W>(st + ST_INV * C, inv);
        load_plane<W>(co + CO_K1 * C, k1);
        load_plane<W>(co + CO_K2 * C, k2);
        load_plane<W>(co + CO_K3 * C, k3);
    } else {
        xv[0] = to_f32<T>(x[e]);
        g[0] = to_f32<T>(dy[e]);
        mean[0] = st[ST_MEAN * C];
        inv[0] = st[ST_INV * C];
        k1[0] = co[CO_K1 * C];
        k2[0] = co[CO_K2 * C];
        k3[0] = co[CO_K3 * C];
    }
#pragma unroll
    for (int k = 0; k < W; ++k) {
        const float xh = (xv[k] - mean[k]) * inv[k];
        g[k] = k1[k] * ((g[k] - k2[k]) - xh * k3[k]);
        if (!mask_pass<T>(mask, mask_f32, e + k)) g[k] = 0.f;
    }
    if constexpr (W > 1) store_vec<T, W>(dx + e, g);
    else dx[e] = from_f32<T>(g[0]);
}

static bool bn_vec(int C, size_t es)
{
    const int v = (int)(16 / es);
    return C % v == 0 && C / v <= 256;
}

// Splits of a shard's rows: enough blocks to fill the GPU (about 1024 over the R shards), at
// least 16 rows per row lane.
static int bn_splits(int R, int C, long long M, size_t es)
{
    const int W = bn_vec(C, es) ? (int)(16 / es) : 1;
    const int G = (C + W - 1) / W;
    const long long lanes = 256 / (G > 256 ? 256 : G);
    long long s = (1024 + R - 1) / R;
    const long long smax = M / (16 * lanes);
    if (s > smax) s = smax;
    return (int)(s < 1 ? 1 : s);
}

size_t bn_partial_doubles(Dt dt, int R, int C, int Nb, int HW)
{
    const size_t es = dt == DT_F32 ? 4 : 2;
    return (size_t)R * bn_splits(R, C, (long long)Nb * HW, es) * C * 2;
}

template <typename T>
static hipError_t bn_fwd_t(int R, int Nb, int HW, int C, const void* x, void* y,
                           const float* gamma, const float* beta, double* part, float* stats,
                           bool relu, hipStream_t s, const void* skip, void* z, bool relu2)
{
    const T* sk = static_cast<const T*>(skip);
    T* zt = static_cast<T*>(z);
    constexpr int V = 16 / sizeof(T);
    const long long M = (long long)Nb * HW;
    const int S = bn_splits(R, C, M, sizeof(T));
    const bool vec = bn_vec(C, sizeof(T));
    if (!vec && C > 256) return hipErrorInvalidValue;  // one block covers every channel
    const T* xt = static_cast<const T*>(x);
    if (vec)
        hipLaunchKernelGGL((bn_partial_kernel<T, false, V>), dim3(S, R), dim3(256),
                           2 * 256 * V * sizeof(double), s, xt, nullptr, nullptr, Nb, HW, C, S,
                           part);
    else
        hipLaunchKernelGGL((bn_partial_kernel<T, false, 1>), dim3(S, R), dim3(256),
                           2 * 256 * sizeof(double), s, xt, nullptr, nullptr, Nb, HW, C, S, part);
    timing_split(s, "finalize");
    hipLaunchKernelGGL((bn_finalize_kernel<false>), dim3((C + 63) / 64, R), dim3(256), 0, s, part,
                       C, S, M, kBnEps, gamma, beta, stats, nullptr, 0ll, 0ll, 0ll, nullptr);
    timing_split(s, "apply");
    const size_t total = (size_t)M * R * C;
    if (vec) {
        const unsigned n = (unsigned)(total / V);
        hipLaunchKernelGGL((bn_apply_kernel<T, V>), dim3((n + 255) / 256), dim3(256), 0, s, xt,
                           static_cast<T*>(y), stats, (unsigned)M, C, n, relu ? 1 : 0, sk, zt,
                           relu2 ? 1 : 0);
    } else {
        const unsigned n = (unsigned)total;
        hipLaunchKernelGGL((bn_apply_kernel<T, 1>), dim3((n + 255) / 256), dim3(256), 0, s, xt,
                           static_cast<T*>(y), stats, (unsigned)M, C, n, relu ? 1 : 0, sk, zt,
                           relu2 ? 1 : 0);
    }
    return hipGetLastError();
}

hipError_t bn_fwd(Dt dt, int R, int Nb, int HW, int C, const void* x, void* y,
                  const float* gamma, const float* beta, double* part, float* stats, bool relu,
                  hipStream_t s, const void* skip, void* z, bool relu2)
{
    if (dt == DT_F32)
        return bn_fwd_t<float>(R, Nb, HW, C, x, y, gamma, beta, part, stats, relu, s, skip, z,
                               relu2);
    return bn_fwd_t<bf16_t>(R, Nb, HW, C, x, y, gamma, beta, part, stats, relu, s, skip, z,
                            relu2);
}

template <typename T>
static hipError_t bn_bwd_t(int R, int Nb, int HW, int C, const void* x, const void* dy, void* dx,
                           const void* mask, bool mask_f32, const float* stats, double* part,
                           float* coef, float* grads, long long ld, long long w_off,
                           long long b_off, hipStream_t s)
{
    constexpr int V = 16 / sizeof(T);
    const long long M = (long long)Nb * HW;
    const int S = bn_splits(R, C, M, sizeof(T));
    const bool vec = bn_vec(C, sizeof(T));
    if (!vec && C > 256) return hipErrorInvalidValue;
    const T* xt = static_cast<const T*>(x);
    const T* gt = static_cast<const T*>(dy);
    if (vec)
        hipLaunchKernelGGL((bn_partial_kernel<T, true, V>), dim3(S, R), dim3(256),
                           2 * 256 * V * sizeof(double), s, xt, gt, stats, Nb, HW, C, S, part);
    else
        hipLaunchKernelGGL((bn_partial_kernel<T, true, 1>), dim3(S, R), dim3(256),
                           2 * 256 * sizeof(double), s, xt, gt, stats, Nb, HW, C, S, part);
    timing_split(s, "finalize");
    hipLaunchKernelGGL((bn_finalize_kernel<true>), dim3((C + 63) / 64, R), dim3(256), 0, s, part,
                       C, S, M, kBnEps, nullptr, nullptr, const_cast<float*>(stats), grads, ld,
                       w_off, b_off, coef);  // read-only in the backward instance
    if (!dx) return hipGetLastError();
    timing_split(s, "apply");
    const size_t total = (size_t)M * R * C;
    if (vec) {
        const unsigned n = (unsigned)(total / V);
        hipLaunchKernelGGL((bn_bwd_apply_kernel<T, V>), dim3((n + 255) / 256), dim3(256), 0, s,
                           xt, gt, stats, coef, mask, mask_f32 ? 1 : 0, static_cast<T*>(dx),
                           (unsigned)M, C, n);
    } else {
        const unsigned n = (unsigned)total;
        hipLaunchKernelGGL((bn_bwd_apply_kernel<T, 1>), dim3((n + 255) / 256), dim3(256), 0, s,
                           xt, gt, stats, coef, mask, mask_f32 ? 1 : 0, static_cast<T*>(dx),
                           (unsigned)M, C, n);
    }
    return hipGetLastError();
}

hipError_t bn_bwd(Dt dt, int R, int Nb, int HW, int C, const void* x, const void* dy, void* dx,
                  const void* mask, bool mask_f32, const float* stats, double* part, float* coef,
                  float* grads, long long ld, long long w_off, long long b_off, hipStream_t s)
{
    if (dt == DT_F32)
        return bn_bwd_t<float>(R, Nb, HW, C, x, dy, dx, mask, mask_f32, stats, part, coef, grads,
                               ld, w_off, b_off, s);
    return bn_bwd_t<bf16_t>(R, Nb, HW, C, x, dy, dx, mask, mask_f32, stats, part, coef, grads, ld,
                            w_off, b_off, s);
}

// ---- residual addition ------------------------------------------------------------------------

template <typename T>
__global__ __launch_bounds__(256) void add_fwd_kernel(const T* __restrict__ a,
                                                      const T* __restrict__ b,
                                                      T* __restrict__ y, unsigned total,
                                                      int relu)
{
    const unsigned t = blockIdx.x * 256 + threadIdx.x;
    if (t >= total) return;
    float v = to_f32<T>(a[t]) + to_f32<T>(b[t]);
    if (relu) v = fmaxf(v, 0.f);
    y[t] = from_f32<T>(v);
}

// The output gradient reaches the previous layer (dx, masked by its ReLU) and the source layer
// (skip, masked by the source's ReLU) unchanged.
template <typename T>
__global__ __launch_bounds__(256) void add_bwd_kernel(const T* __restrict__ dy,
                                                      T* __restrict__ dx, const void* mask,
                                                      int mask_f32, T* __restrict__ skip,
                                                      const void* smask, int smask_f32,
                                                      unsigned total)
{
    const unsigned t = blockIdx.x * 256 + threadIdx.x;
    if (t >= total) return;
    const T g = dy[t];
    if (dx) dx[t] = mask_pass<T>(mask, mask_f32, t) ? g : from_f32<T>(0.f);
    if (skip) skip[t] = mask_pass<T>(smask, smask_f32, t) ? g : from_f32<T>(0.f);
}

// dy += skip where the source's ReLU passed (smask: its stored output; null: everywhere)
template <typename T>
__global__ __launch_bounds__(256) void skip_add_kernel(T* __restrict__ dy,
                                                       const T* __restrict__ skip,
                                                       const void* smask, int smask_f32,
                                                       unsigned total)
{
    const unsigned t = blockIdx.x * 256 + threadIdx.x;
    if (t >= total) return;
    const float g = mask_pass<T>(smask, smask_f32, t) ? to_f32<T>(skip[t]) : 0.f;
    dy[t] = from_f32<T>(to_f32<T>(dy[t]) + g);
}

// 16-byte variants: V consecutive elements per thread (n a multiple of V).
template <typename T>
__global__ __launch_bounds__(256) void add_fwd_vec_kernel(const T* __restrict__ a,
                                                          const T* __restrict__ b,
                                                          T* __restrict__ y, unsigned nvec,
                                                          int relu)
{
    constexpr int V = 16 / sizeof(T);
    const unsigned t = blockIdx.x * 256 + threadIdx.x;
    if (t >= nvec) return;
    float va[V], vb[V];
    load_vec<T, V>(a + (size_t)t * V, va);
    load_vec<T, V>(b + (size_t)t * V, vb);
#pragma unroll
    for (int k = 0; k < V; ++k) {
        va[k] += vb[k];
        if (relu) va[k] = fmaxf(va[k], 0.f);
    }
    store_vec<T, V>(y + (size_t)t * V, va);
}

template <typename T, int V>
__device__ __forceinline__ void load_mask(const void* m, int m_f32, size_t e, float (&v)[V])
{
    if (!m) {
#pragma unroll
        for (int k = 0; k < V; ++k) v[k] = 1.f;
    } else if (m_f32) {
#pragma unroll
        for (int k = 0; k < V; ++k) v[k] = static_cast<const float*>(m)[e + k];
    } else {
        load_vec<T, V>(static_cast<const T*>(m) + e, v);
    }
}

template <typename T>
__global__ __launch_bounds__(256) void add_bwd_vec_kernel(const T* __restrict__ dy,
                                                          T* __restrict__ dx, const void* mask,
                                                          int mask_f32, T* __restrict__ skip,
                                                          const void* smask, int smask_f32,
                                                          unsigned nvec)
{
    constexpr int V = 16 / sizeof(T);
    const unsigned t = blockIdx.x * 256 + threadIdx.x;
    if (t >= nvec) return;
    const size_t e = (size_t)t * V;
    float g[V], m[V], o[V];
    load_vec<T, V>(dy + e, g);
    if (dx) {
        load_mask<T, V>(mask, mask_f32, e, m);
#pragma unroll
        for (int k = 0; k < V; ++k) o[k] = m[k] > 0.f ? g[k] : 0.f;
        store_vec<T, V>(dx + e, o);
    }
    if (skip) {
        load_mask<T, V>(smask, smask_f32, e, m);
#pragma unroll
        for (int k = 0; k < V; ++k) o[k] = m[k] > 0.f ? g[k] : 0.f;
        store_vec<T, V>(skip + e, o);
    }
}

template <typename T>
__global__ __launch_bounds__(256) void skip_add_vec_kernel(T* __restrict__ dy,
                                                           const T* __restrict__ skip,
                                                           const void* smask, int smask_f32,
                                                           unsigned nvec)
{
    constexpr int V = 16 / sizeof(T);
    const unsigned t = blockIdx.x * 256 + threadIdx.x;
    if (t >= nvec) return;
    const size_t e = (size_t)t * V;
    float a[V], b[V], m[V];
    load_vec<T, V>(dy + e, a);
    load_vec<T, V>(skip + e, b);
    load_mask<T, V>(smask, smask_f32, e, m);
#pragma unroll
    for (int k = 0; k < V; ++k) a[k] += m[k] > 0.f ? b[k] : 0.f;
    store_vec<T, V>(dy + e, a);
}

hipError_t add_fwd(Dt dt, size_t n, const void* a, const void* b, void* y, bool relu,
                   hipStream_t s)
{
    const size_t V = dt == DT_F32 ? 4 : 8;
    if (n % V == 0) {
        const unsigned nv = (unsigned)(n / V);
        const dim3 g((nv + 255) / 256);
        if (dt == DT_F32)
            hipLaunchKernelGGL((add_fwd_vec_kernel<float>), g, dim3(256), 0, s,
                               static_cast<const float*>(a), static_cast<const float*>(b),
                               static_cast<float*>(y), nv, relu ? 1 : 0);
        else
            hipLaunchKernelGGL((add_fwd_vec_kernel<bf16_t>), g, dim3(256), 0, s,
                               static_cast<const bf16_t*>(a), static_cast<const bf16_t*>(b),
                               static_cast<bf16_t*>(y), nv, relu ? 1 : 0);
        return hipGetLastError();
    }
    const unsigned total = (unsigned)n;
    const dim3 g((total + 255) / 256);
    if (dt == DT_F32)
        hipLaunchKernelGGL((add_fwd_kernel<float>), g, dim3(256), 0, s,
                           static_cast<const float*>(a), static_cast<const float*>(b),
                           static_cast<float*>(y), total, relu ? 1 : 0);
    else
        hipLaunchKernelGGL((add_fwd_kernel<bf16_t>), g, dim3(256), 0, s,
                           static_cast<const bf16_t*>(a), static_cast<const bf16_t*>(b),
                           static_cast<bf16_t*>(y), total, relu ? 1 : 0);
    return hipGetLastError();
}

hipError_t add_bwd(Dt dt, size_t n, const void* dy, void* dx, const void* mask, bool mask_f32,
                   void* skip, const void* smask, bool smask_f32, hipStream_t s)
{
    const size_t V = dt == DT_F32 ? 4 : 8;
    if (n % V == 0) {
        const unsigned nv = (unsigned)(n / V);
        const dim3 g((nv + 255) / 256);
        if (dt == DT_F32)
            hipLaunchKernelGGL((add_bwd_vec_kernel<float>), g, dim3(256), 0, s,
                               static_cast<const float*>(dy), static_cast<float*>(dx), mask,
                               mask_f32 ? 1 : 0, static_cast<float*>(skip), smask,
                               smask_f32 ? 1 : 0, nv);
        else
            hipLaunchKernelGGL((add_bwd_vec_kernel<bf16_t>), g, dim3(256), 0, s,
                               static_cast<const bf16_t*>(dy), static_cast<bf16_t*>(dx), mask,
                               mask_f32 ? 1 : 0, static_cast<bf16_t*>(skip), smask,
                               smask_f32 ? 1 : 0, nv);
        return hipGetLastError();
    }
    const unsigned total = (unsigned)n;
    const dim3 g((total + 255) / 256);
    if (dt == DT_F32)
        hipLaunchKernelGGL((add_bwd_kernel<float>), g, dim3(256), 0, s,
                           static_cast<const float*>(dy), static_cast<float*>(dx), mask,
                           mask_f32 ? 1 : 0, static_cast<float*>(skip), smask,
                           smask_f32 ? 1 : 0, total);
    else
        hipLaunchKernelGGL((add_bwd_kernel<bf16_t>), g, dim3(256), 0, s,
                           static_cast<const bf16_t*>(dy), static_cast<bf16_t*>(dx), mask,
                           mask_f32 ? 1 : 0, static_cast<bf16_t*>(skip), smask,
                           smask_f32 ? 1 : 0, total);
    return hipGetLastError();
}

hipError_t skip_add(Dt dt, size_t n, void* dy, const void* skip, const void* smask,
                    bool smask_f32, hipStream_t s)
{
    const size_t V = dt == DT_F32 ? 4 : 8;
    const int mf = smask_f32 ? 1 : 0;
    if (n % V == 0) {
        const unsigned nv = (unsigned)(n / V);
        const dim3 g((nv + 255) / 256);
        if (dt == DT_F32)
            hipLaunchKernelGGL((skip_add_vec_kernel<float>), g, dim3(256), 0, s,
                               static_cast<float*>(dy), static_cast<const float*>(skip), smask,
                               mf, nv);
        else
            hipLaunchKernelGGL((skip_add_vec_kernel<bf16_t>), g, dim3(256), 0, s,
                               static_cast<bf16_t*>(dy), static_cast<const bf16_t*>(skip), smask,
                               mf, nv);
        return hipGetLastError();
    }
    const unsigned total = (unsigned)n;
    const dim3 g((total + 255) / 256);
    if (dt == DT_F32)
        hipLaunchKernelGGL((skip_add_kernel<float>), g, dim3(256), 0, s, static_cast<float*>(dy),
                           static_cast<const float*>(skip), smask, mf, total);
    else
        hipLaunchKernelGGL((skip_add_kernel<bf16_t>), g, dim3(256), 0, s,
                           static_cast<bf16_t*>(dy), static_cast<const bf16_t*>(skip), smask, mf,
                           total);
    return hipGetLastError();
}

}  // namespace mtx
