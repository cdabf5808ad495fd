// Batch normalisation with per-shard statistics and the residual addition (the building blocks
// of the ResNet-50 network in Table II), over NHWC tensors [R*Nb][H*W][C] of all R shards.
//
// Batch normalisation normalises channel c of shard r by the mean and the biased variance of
// its M = Nb*H*W values: y = gamma (x - mean) / sqrt(var + eps) + beta.  The per-shard sums are
// reductions over rows: blocks of 64 channels x 4 row lanes take a contiguous range of the
// shard's rows (one of S splits), add in double, and write one partial per (shard, split,
// channel); a finalize kernel adds the S partials in ascending order.  No atomics: results are
// the same on every run.
#include "device_common.h"
#include "internal.h"

namespace mtx {

constexpr int kBnCh = 64;  // channels per reduction block (one per lane of a wave)

// A ReLU mask read from the stored output of a layer (fp32 or the compute type).
template <typename T>
__device__ __forceinline__ bool mask_pass(const void* m, int m_f32, unsigned t)
{
    if (!m) return true;
    const float v = m_f32 ? static_cast<const float*>(m)[t] : to_f32<T>(static_cast<const T*>(m)[t]);
    return v > 0.f;
}

// Row sums of shard r = blockIdx.z, split s = blockIdx.y, channels blockIdx.x*64 + lane.
//   forward:  (sum x, sum x^2)
//   backward: (sum dy, sum dy * xhat) with xhat = (x - mean) * inv from `stats`
template <typename T, bool BWD>
__global__ __launch_bounds__(256) void bn_partial_kernel(const T* __restrict__ x,
                                                         const T* __restrict__ dy,
                                                         const float* __restrict__ stats, int Nb,
                                                         int HW, int C, int S,
                                                         double* __restrict__ part)
{
    const int lane = threadIdx.x & 63, q = threadIdx.x >> 6;
    const int c = blockIdx.x * kBnCh + lane, s = blockIdx.y, r = blockIdx.z;
    const long long M = (long long)Nb * HW;
    const long long per = (M + S - 1) / S;
    const long long r0 = (long long)s * per, r1 = min(M, r0 + per);
    double a = 0.0, b = 0.0;
    if (c < C) {
        const long long base = (long long)r * M;
        float mean = 0.f, inv = 0.f;
        if (BWD) {
            mean = stats[((long long)r * C + c) * 2];
            inv = stats[((long long)r * C + c) * 2 + 1];
        }
        for (long long i = r0 + q; i < r1; i += 4) {
            const long long o = (base + i) * C + c;
            const float xv = to_f32<T>(x[o]);
            if (!BWD) {
                a += (double)xv;
                b += (double)xv * (double)xv;
            } else {
                const float g = to_f32<T>(dy[o]);
                a += (double)g;
                b += (double)g * (double)((xv - mean) * inv);
            }
        }
    }
    __shared__ double sa[4][kBnCh], sb[4][kBnCh];
    sa[q][lane] = a;
    sb[q][lane] = b;
    __syncthreads();
    if (q == 0 && c < C) {
        double* p = part + (((long long)r * S + s) * C + c) * 2;
        p[0] = ((sa[0][lane] + sa[1][lane]) + sa[2][lane]) + sa[3][lane];
        p[1] = ((sb[0][lane] + sb[1][lane]) + sb[2][lane]) + sb[3][lane];
    }
}

// Forward statistics per (shard, channel): mean and 1 / sqrt(var + eps), var = E[x^2] - mean^2
// in double (the sums are double, so the cancellation costs nothing at these sizes).
__global__ __launch_bounds__(256) void bn_stats_kernel(const double* __restrict__ part, int R,
                                                       int C, int S, long long M, double eps,
                                                       float* __restrict__ stats)
{
    const int t = blockIdx.x * 256 + threadIdx.x;
    if (t >= R * C) return;
    const int r = t / C, c = t - r * C;
    double a = 0.0, b = 0.0;
    for (int s = 0; s < S; ++s) {
        const double* p = part + (((long long)r * S + s) * C + c) * 2;
        a += p[0];
        b += p[1];
    }
    const double mean = a / (double)M;
    const double var = fmax(b / (double)M - mean * mean, 0.0);
    stats[(long long)t * 2] = (float)mean;
    stats[(long long)t * 2 + 1] = (float)(1.0 / sqrt(var + eps));
}

// y = gamma * (x - mean) * inv + beta, ReLU, stored in the compute type.
template <typename T>
__global__ __launch_bounds__(256) void bn_apply_kernel(const T* __restrict__ x, T* __restrict__ y,
                                                       const float* __restrict__ gamma,
                                                       const float* __restrict__ beta,
                                                       const float* __restrict__ stats,
                                                       unsigned rows_per_shard, int C,
                                                       unsigned total, int relu)
{
    const unsigned t = blockIdx.x * 256 + threadIdx.x;
    if (t >= total) return;
    const unsigned row = t / (unsigned)C, c = t - row * (unsigned)C;
    const unsigned r = row / rows_per_shard;
    const float* st = stats + ((size_t)r * C + c) * 2;
    float v = fmaf(gamma[c], (to_f32<T>(x[t]) - st[0]) * st[1], beta[c]);
    if (relu) v = fmaxf(v, 0.f);
    y[t] = from_f32<T>(v);
}

// Backward per (shard, channel): the shard's gamma and beta gradients (rows of grads) and the
// coefficients of dx = k1 * (dy - k2 - xhat * k3), k1 = gamma * inv, k2 = sum dy / M,
// k3 = sum(dy xhat) / M.
__global__ __launch_bounds__(256) void bn_bwd_coef_kernel(const double* __restrict__ part,
                                                          const float* __restrict__ gamma,
                                                          const float* __restrict__ stats, int R,
                                                          int C, int S, long long M,
                                                          float* __restrict__ grads,
                                                          long long ld, long long w_off,
                                                          long long b_off,
                                                          float* __restrict__ coef)
{
    const int t = blockIdx.x * 256 + threadIdx.x;
    if (t >= R * C) return;
    const int r = t / C, c = t - r * C;
    double sd = 0.0, sdx = 0.0;
    for (int s = 0; s < S; ++s) {
        const double* p = part + (((long long)r * S + s) * C + c) * 2;
        sd += p[0];
        sdx += p[1];
    }
    grads[(long long)r * ld + w_off + c] = (float)sdx;
    grads[(long long)r * ld + b_off + c] = (float)sd;
    coef[(long long)t * 3] = gamma[c] * stats[(long long)t * 2 + 1];
    coef[(long long)t * 3 + 1] = (float)(sd / (double)M);
    coef[(long long)t * 3 + 2] = (float)(sdx / (double)M);
}

template <typename T>
__global__ __launch_bounds__(256) void bn_bwd_apply_kernel(
    const T* __restrict__ x, const T* __restrict__ dy, const float* __restrict__ stats,
    const float* __restrict__ coef, const void* mask, int mask_f32, T* __restrict__ dx,
    unsigned rows_per_shard, int C, unsigned total)
{
    const unsigned t = blockIdx.x * 256 + threadIdx.x;
    if (t >= total) return;
    const unsigned row = t / (unsigned)C, c = t - row * (unsigned)C;
    const size_t rc = (size_t)(row / rows_per_shard) * C + c;
    const float xh = (to_f32<T>(x[t]) - stats[rc * 2]) * stats[rc * 2 + 1];
    const float* k = coef + rc * 3;
    float v = k[0] * ((to_f32<T>(dy[t]) - k[1]) - xh * k[2]);
    if (!mask_pass<T>(mask, mask_f32, t)) v = 0.f;
    dx[t] = from_f32<T>(v);
}

static int bn_splits(long long M)
{
    long long s = M / 2048;
    return (int)(s < 1 ? 1 : (s > 64 ? 64 : s));
}

size_t bn_partial_doubles(int R, int C, int Nb, int HW)
{
    return (size_t)R * bn_splits((long long)Nb * HW) * C * 2;
}

template <typename T>
static hipError_t bn_fwd_t(int R, int Nb, int HW, int C, const void* x, void* y,
                           const float* gamma, const float* beta, double* part, float* stats,
                           bool relu, hipStream_t s)
{
    const long long M = (long long)Nb * HW;
    const int S = bn_splits(M);
    hipLaunchKernelGGL((bn_partial_kernel<T, false>), dim3((C + kBnCh - 1) / kBnCh, S, R),
                       dim3(256), 0, s, static_cast<const T*>(x), nullptr, nullptr, Nb, HW, C,
                       S, part);
    hipLaunchKernelGGL(bn_stats_kernel, dim3((R * C + 255) / 256), dim3(256), 0, s, part, R, C, S,
                       M, kBnEps, stats);
    timing_split(s, "apply");
    const unsigned total = (unsigned)(M * R * C);
    hipLaunchKernelGGL((bn_apply_kernel<T>), dim3((total + 255) / 256), dim3(256), 0, s,
                       static_cast<const T*>(x), static_cast<T*>(y), gamma, beta, stats,
                       (unsigned)M, C, total, relu ? 1 : 0);
    return hipGetLastError();
}

hipError_t bn_fwd(Dt dt, int R, int Nb, int HW, int C, const void* x, void* y,
                  const float* gamma, const float* beta, double* part, float* stats, bool relu,
                  hipStream_t s)
{
    if (dt == DT_F32) return bn_fwd_t<float>(R, Nb, HW, C, x, y, gamma, beta, part, stats, relu, s);
    return bn_fwd_t<bf16_t>(R, Nb, HW, C, x, y, gamma, beta, part, stats, relu, s);
}

template <typename T>
static hipError_t bn_bwd_t(int R, int Nb, int HW, int C, const void* x, const void* dy, void* dx,
                           const void* mask, bool mask_f32, const float* gamma,
                           const float* stats, double* part, float* coef, float* grads,
                           long long ld, long long w_off, long long b_off, hipStream_t s)
{
    const long long M = (long long)Nb * HW;
    const int S = bn_splits(M);
    hipLaunchKernelGGL((bn_partial_kernel<T, true>), dim3((C + kBnCh - 1) / kBnCh, S, R),
                       dim3(256), 0, s, static_cast<const T*>(x), static_cast<const T*>(dy),
                       stats, Nb, HW, C, S, part);
    hipLaunchKernelGGL(bn_bwd_coef_kernel, dim3((R * C + 255) / 256), dim3(256), 0, s, part,
                       gamma, stats, R, C, S, M, grads, ld, w_off, b_off, coef);
    if (!dx) return hipGetLastError();
    timing_split(s, "apply");
    const unsigned total = (unsigned)(M * R * C);
    hipLaunchKernelGGL((bn_bwd_apply_kernel<T>), dim3((total + 255) / 256), dim3(256), 0, s,
                       static_cast<const T*>(x), static_cast<const T*>(dy), stats, coef, mask,
                       mask_f32 ? 1 : 0, static_cast<T*>(dx), (unsigned)M, C, total);
    return hipGetLastError();
}

hipError_t bn_bwd(Dt dt, int R, int Nb, int HW, int C, const void* x, const void* dy, void* dx,
                  const void* mask, bool mask_f32, const float* gamma, const float* stats,
                  double* part, float* coef, float* grads, long long ld, long long w_off,
                  long long b_off, hipStream_t s)
{
    if (dt == DT_F32)
        return bn_bwd_t<float>(R, Nb, HW, C, x, dy, dx, mask, mask_f32, gamma, stats, part, coef,
                               grads, ld, w_off, b_off, s);
    return bn_bwd_t<bf16_t>(R, Nb, HW, C, x, dy, dx, mask, mask_f32, gamma, stats, part, coef,
                            grads, ld, w_off, b_off, s);
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

template <typename T>
__global__ __launch_bounds__(256) void skip_add_kernel(T* __restrict__ dy,
                                                       const T* __restrict__ skip,
                                                       unsigned total)
{
    const unsigned t = blockIdx.x * 256 + threadIdx.x;
    if (t >= total) return;
    dy[t] = from_f32<T>(to_f32<T>(dy[t]) + to_f32<T>(skip[t]));
}

hipError_t add_fwd(Dt dt, size_t n, const void* a, const void* b, void* y, bool relu,
                   hipStream_t s)
{
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

hipError_t skip_add(Dt dt, size_t n, void* dy, const void* skip, hipStream_t s)
{
    const unsigned total = (unsigned)n;
    const dim3 g((total + 255) / 256);
    if (dt == DT_F32)
        hipLaunchKernelGGL((skip_add_kernel<float>), g, dim3(256), 0, s, static_cast<float*>(dy),
                           static_cast<const float*>(skip), total);
    else
        hipLaunchKernelGGL((skip_add_kernel<bf16_t>), g, dim3(256), 0, s,
                           static_cast<bf16_t*>(dy), static_cast<const bf16_t*>(skip), total);
    return hipGetLastError();
}

}  // namespace mtx
