// Memory-bound kernels of the training step: bfloat16 casts, max-pooling, the fused softmax
// cross-entropy and the fused gradient average + momentum update.  All reductions run in a fixed order, so results
// are identical from run to run.
#include "device_common.h"
#include "internal.h"

namespace mtx {

static inline unsigned grid_for(size_t n, unsigned per_block)
{
    size_t g = (n + per_block - 1) / per_block;
    return (unsigned)(g ? g : 1);
}

// ---- fp32 -> bfloat16 (round to nearest even), 4 elements per thread ------------------------

__global__ __launch_bounds__(256) void cast_bf16_kernel(const float* __restrict__ src,
                                                        bf16_t* __restrict__ dst, size_t n)
{
    const size_t i = ((size_t)blockIdx.x * 256 + threadIdx.x) * 4;
    if (i + 3 < n && ((reinterpret_cast<uintptr_t>(src + i) & 15) == 0)) {
        const float4 f = *reinterpret_cast<const float4*>(src + i);
        const uint32_t lo = f32_to_bf16(f.x) | ((uint32_t)f32_to_bf16(f.y) << 16);
        const uint32_t hi = f32_to_bf16(f.z) | ((uint32_t)f32_to_bf16(f.w) << 16);
        if ((reinterpret_cast<uintptr_t>(dst + i) & 7) == 0) {
            *reinterpret_cast<uint2*>(dst + i) = make_uint2(lo, hi);
            return;
        }
    }
    for (size_t j = i; j < i + 4 && j < n; ++j) dst[j] = f32_to_bf16(src[j]);
}

hipError_t cast_bf16(const float* src, void* dst, size_t n, hipStream_t s)
{
    if (!n) return hipSuccess;
    hipLaunchKernelGGL(cast_bf16_kernel, dim3(grid_for(n, 1024)), dim3(256), 0, s, src,
                       static_cast<bf16_t*>(dst), n);
    return hipGetLastError();
}

// ---- max-pooling ----------------------------------------------------------------------------

// One thread per output: the first maximal element of the K x K window in row-major order.
template <typename T>
__global__ __launch_bounds__(256) void pool_fwd_kernel(int total, int H, int W, int K, int S,
                                                       int OH, int OW, const T* __restrict__ x,
                                                       T* __restrict__ y,
                                                       uint8_t* __restrict__ argmax)
{
    const int o = blockIdx.x * 256 + threadIdx.x;
    if (o >= total) return;
    const int ohw = OH * OW;
    const int nc = o / ohw, hw = o - nc * ohw, i = hw / OW, j = hw - i * OW;
    const T* xp = x + (long long)nc * H * W + (long long)(i * S) * W + j * S;
    T best = xp[0];
    float bv = to_f32<T>(best);
    int bi = 0;
    for (int u = 0; u < K; ++u)
        for (int v = 0; v < K; ++v) {
            const T t = xp[u * W + v];
            const float tv = to_f32<T>(t);
            if (tv > bv) { bv = tv; best = t; bi = u * K + v; }
        }
    y[o] = best;
    argmax[o] = (uint8_t)bi;
}

hipError_t pool_fwd(Dt dt, int N, int C, int H, int W, int K, int S, const void* x, void* y,
                    uint8_t* argmax, hipStream_t s)
{
    const int OH = (H - K) / S + 1, OW = (W - K) / S + 1;
    const int total = N * C * OH * OW;
    if (total <= 0) return hipSuccess;
    if (dt == DT_F32)
        hipLaunchKernelGGL(pool_fwd_kernel<float>, dim3(grid_for(total, 256)), dim3(256), 0, s,
                           total, H, W, K, S, OH, OW, static_cast<const float*>(x),
                           static_cast<float*>(y), argmax);
    else
        hipLaunchKernelGGL(pool_fwd_kernel<bf16_t>, dim3(grid_for(total, 256)), dim3(256), 0, s,
                           total, H, W, K, S, OH, OW, static_cast<const bf16_t*>(x),
                           static_cast<bf16_t*>(y), argmax);
    return hipGetLastError();
}

// One thread per input element: the sum, in ascending window order, of the output gradients
// of the windows whose maximum sits here (windows overlap when S < K), times the ReLU mask of
// the layer that produced the pooled tensor.  Gathering keeps the result free of atomics.
template <typename T>
__global__ __launch_bounds__(256) void pool_bwd_kernel(int total, int H, int W, int K, int S,
                                                       int OH, int OW,
                                                       const uint8_t* __restrict__ argmax,
                                                       const T* __restrict__ dy,
                                                       T* __restrict__ dx,
                                                       const void* __restrict__ mask,
                                                       int mask_f32)
{
    const int t = blockIdx.x * 256 + threadIdx.x;
    if (t >= total) return;
    const int hw_in = H * W;
    const int nc = t / hw_in, hw = t - nc * hw_in, h = hw / W, w = hw - h * W;
    // windows i with i*S <= h <= i*S + K - 1
    const int ilo = h - K + 1 <= 0 ? 0 : (h - K + 1 + S - 1) / S;
    const int ihi = min(h / S, OH - 1);
    const int jlo = w - K + 1 <= 0 ? 0 : (w - K + 1 + S - 1) / S;
    const int jhi = min(w / S, OW - 1);
    float acc = 0.f;
    const long long base = (long long)nc * OH * OW;
    for (int i = ilo; i <= ihi; ++i)
        for (int j = jlo; j <= jhi; ++j) {
            const long long o = base + (long long)i * OW + j;
            const int here = (h - i * S) * K + (w - j * S);
            if (argmax[o] == here) acc += to_f32<T>(dy[o]);
        }
    if (mask) {
        const float m = mask_f32 ? static_cast<const float*>(mask)[t]
                                 : to_f32<T>(static_cast<const T*>(mask)[t]);
        if (!(m > 0.f)) acc = 0.f;
    }
    dx[t] = from_f32<T>(acc);
}

hipError_t pool_bwd(Dt dt, int N, int C, int H, int W, int K, int S, const uint8_t* argmax,
                    const void* dy, void* dx, const void* mask, bool mask_f32, hipStream_t s)
{
    const int OH = (H - K) / S + 1, OW = (W - K) / S + 1;
    const int total = N * C * H * W;
    if (total <= 0) return hipSuccess;
    if (dt == DT_F32)
        hipLaunchKernelGGL(pool_bwd_kernel<float>, dim3(grid_for(total, 256)), dim3(256), 0, s,
                           total, H, W, K, S, OH, OW, argmax, static_cast<const float*>(dy),
                           static_cast<float*>(dx), mask, (int)mask_f32);
    else
        hipLaunchKernelGGL(pool_bwd_kernel<bf16_t>, dim3(grid_for(total, 256)), dim3(256), 0, s,
                           total, H, W, K, S, OH, OW, argmax, static_cast<const bf16_t*>(dy),
                           static_cast<bf16_t*>(dx), mask, (int)mask_f32);
    return hipGetLastError();
}

// ---- softmax cross-entropy ------------------------------------------------------------------

__device__ __forceinline__ float wave_max(float v)
{
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
    return v;
}

__device__ __forceinline__ float wave_sum(float v)
{
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

// One wave per sample: loss = logsumexp(z) - z[y] with the row maximum subtracted, and
// dz = (softmax(z) - onehot(y)) / Nb (the gradient of the shard-mean loss), stored in the
// compute type.
template <typename T>
__global__ __launch_bounds__(256) void softmax_xent_kernel(int B, int NC, float inv_nb,
                                                           const float* __restrict__ z,
                                                           const int32_t* __restrict__ labels,
                                                           float* __restrict__ loss_rows,
                                                           T* __restrict__ dz)
{
    const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (row >= B) return;
    const float* zr = z + (long long)row * NC;
    float m = -INFINITY;
    for (int c = lane; c < NC; c += 64) m = fmaxf(m, zr[c]);
    m = wave_max(m);
    float se = 0.f;
    for (int c = lane; c < NC; c += 64) se += expf(zr[c] - m);
    se = wave_sum(se);
    const float lse = m + logf(se);
    const int y = labels[row];
    const bool valid = y >= 0 && y < NC;
    for (int c = lane; c < NC; c += 64) {
        const float p = expf(zr[c] - lse);
        dz[(long long)row * NC + c] = from_f32<T>((p - (c == y ? 1.f : 0.f)) * inv_nb);
    }
    if (lane == 0) loss_rows[row] = valid ? lse - zr[y] : __int_as_float(0x7fc00000);
}

hipError_t softmax_xent(Dt dt, int B, int NC, int Nb, const float* logits,
                        const int32_t* labels, float* loss_rows, void* dz, hipStream_t s)
{
    const float inv = 1.0f / (float)Nb;
    dim3 grid((B + 3) / 4);
    if (dt == DT_F32)
        hipLaunchKernelGGL(softmax_xent_kernel<float>, grid, dim3(256), 0, s, B, NC, inv, logits,
                           labels, loss_rows, static_cast<float*>(dz));
    else
        hipLaunchKernelGGL(softmax_xent_kernel<bf16_t>, grid, dim3(256), 0, s, B, NC, inv,
                           logits, labels, loss_rows, static_cast<bf16_t*>(dz));
    return hipGetLastError();
}

// Mean of the per-sample losses in a fixed order (one block): the batch-mean loss, which is
// also the mean of the R shard-mean losses since the shards are equal.
__global__ __launch_bounds__(256) void mean_loss_kernel(const float* __restrict__ rows, int B,
                                                        float* __restrict__ out)
{
    __shared__ float sh[256];
    float s = 0.f;
    for (int i = threadIdx.x; i < B; i += 256) s += rows[i];
    sh[threadIdx.x] = s;
    __syncthreads();
    for (int o = 128; o >= 1; o >>= 1) {
        if ((int)threadIdx.x < o) sh[threadIdx.x] += sh[threadIdx.x + o];
        __syncthreads();
    }
    if (threadIdx.x == 0) out[0] = sh[0] / (float)B;
}

hipError_t mean_loss(const float* loss_rows, int B, float* loss_out, hipStream_t s)
{
    hipLaunchKernelGGL(mean_loss_kernel, dim3(1), dim3(256), 0, s, loss_rows, B, loss_out);
    return hipGetLastError();
}

// ---- gradient average + momentum update --------------------------------------------------------
//
// g = (1/R) sum_r grads[r][i] (ascending r, fp32), then v = mu*v + g and w = w - lr*v (each one
// fused multiply-add, i.e. one rounding), or w = w - lr*g without momentum.  Four consecutive
// elements per thread with 16-byte loads when every row is 16-byte aligned; the R loads of a
// thread are independent and issued before the adds.

typedef float f32x4 __attribute__((ext_vector_type(4)));

template <int RT, bool MOM, bool AVG, bool UPD>
__global__ __launch_bounds__(256) void avg_update_vec4(const float* __restrict__ grads, int Rrt,
                                                       long long n4, long long ld,
                                                       float* __restrict__ w,
                                                       float* __restrict__ v, float lr, float mu,
                                                       float* __restrict__ avg)
{
    const long long t = (long long)blockIdx.x * 256 + threadIdx.x;
    if (t >= n4) return;
    const int R = RT > 0 ? RT : Rrt;
    const f32x4* g4 = reinterpret_cast<const f32x4*>(grads) + t;
    const long long ld4 = ld / 4;
    f32x4 s = __builtin_nontemporal_load(g4);
    if (RT > 0) {
        f32x4 buf[RT > 1 ? RT - 1 : 1];
#pragma unroll
        for (int r = 1; r < RT; ++r) buf[r - 1] = __builtin_nontemporal_load(g4 + r * ld4);
#pragma unroll
        for (int r = 1; r < RT; ++r) s += buf[r - 1];
    } else {
        for (int r = 1; r < R; ++r) s += __builtin_nontemporal_load(g4 + r * ld4);
    }
    const float fr = (float)R;
    f32x4 g = {s[0] / fr, s[1] / fr, s[2] / fr, s[3] / fr};
    if (AVG) __builtin_nontemporal_store(g, reinterpret_cast<f32x4*>(avg) + t);
    if (UPD) {
        f32x4 wv = reinterpret_cast<f32x4*>(w)[t];
        if (MOM) {
            f32x4 vv = reinterpret_cast<f32x4*>(v)[t];
#pragma unroll
            for (int j = 0; j < 4; ++j) vv[j] = fmaf(mu, vv[j], g[j]);
            reinterpret_cast<f32x4*>(v)[t] = vv;
            g = vv;
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) wv[j] = fmaf(-lr, g[j], wv[j]);
        reinterpret_cast<f32x4*>(w)[t] = wv;
    }
}

template <bool MOM, bool AVG, bool UPD>
__global__ __launch_bounds__(256) void avg_update_scalar(const float* __restrict__ grads, int R,
                                                         long long n, long long ld,
                                                         float* __restrict__ w,
                                                         float* __restrict__ v, float lr,
                                                         float mu, float* __restrict__ avg)
{
    const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
    if (i >= n) return;
    float s = grads[i];
    for (int r = 1; r < R; ++r) s += grads[(long long)r * ld + i];
    float g = s / (float)R;
    if (AVG) avg[i] = g;
    if (UPD) {
        if (MOM) {
            const float vn = fmaf(mu, v[i], g);
            v[i] = vn;
            g = vn;
        }
        w[i] = fmaf(-lr, g, w[i]);
    }
}

template <bool MOM, bool AVG, bool UPD>
static hipError_t avg_update_launch(const float* grads, int R, size_t n, size_t ld, float* w,
                                    float* v, float lr, float mu, float* avg, hipStream_t s)
{
    auto al = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; };
    const bool vec = (n % 4 == 0) && (ld % 4 == 0) && al(grads) && (!AVG || al(avg)) &&
                     (!UPD || al(w)) && (!MOM || al(v));
    if (vec) {
        const long long n4 = (long long)(n / 4);
        dim3 grid(grid_for(n / 4, 256));
        switch (R) {
        case 1: hipLaunchKernelGGL((avg_update_vec4<1, MOM, AVG, UPD>), grid, dim3(256), 0, s, grads, R, n4, (long long)ld, w, v, lr, mu, avg); break;
        case 2: hipLaunchKernelGGL((avg_update_vec4<2, MOM, AVG, UPD>), grid, dim3(256), 0, s, grads, R, n4, (long long)ld, w, v, lr, mu, avg); break;
        case 4: hipLaunchKernelGGL((avg_update_vec4<4, MOM, AVG, UPD>), grid, dim3(256), 0, s, grads, R, n4, (long long)ld, w, v, lr, mu, avg); break;
        case 8: hipLaunchKernelGGL((avg_update_vec4<8, MOM, AVG, UPD>), grid, dim3(256), 0, s, grads, R, n4, (long long)ld, w, v, lr, mu, avg); break;
        case 16: hipLaunchKernelGGL((avg_update_vec4<16, MOM, AVG, UPD>), grid, dim3(256), 0, s, grads, R, n4, (long long)ld, w, v, lr, mu, avg); break;
        default: hipLaunchKernelGGL((avg_update_vec4<0, MOM, AVG, UPD>), grid, dim3(256), 0, s, grads, R, n4, (long long)ld, w, v, lr, mu, avg); break;
        }
    } else {
        hipLaunchKernelGGL((avg_update_scalar<MOM, AVG, UPD>), dim3(grid_for(n, 256)), dim3(256),
                           0, s, grads, R, (long long)n, (long long)ld, w, v, lr, mu, avg);
    }
    return hipGetLastError();
}

hipError_t average_update(const float* grads, int R, size_t n, size_t ld, float* w, float* v,
                          float lr, float mu, float* avg, bool update, hipStream_t s)
{
    const bool mom = update && mu != 0.0f;
    const bool wavg = avg != nullptr;
    if (!update) return avg_update_launch<false, true, false>(grads, R, n, ld, w, v, lr, mu, avg, s);
    if (mom) {
        if (wavg) return avg_update_launch<true, true, true>(grads, R, n, ld, w, v, lr, mu, avg, s);
        return avg_update_launch<true, false, true>(grads, R, n, ld, w, v, lr, mu, avg, s);
    }
    if (wavg) return avg_update_launch<false, true, true>(grads, R, n, ld, w, v, lr, mu, avg, s);
    return avg_update_launch<false, false, true>(grads, R, n, ld, w, v, lr, mu, avg, s);
}

}  // namespace mtx
