// Memory-bound kernels of the training step: layout conversions and the per-step weight
// preparation, max-pooling, the fused softmax cross-entropy and the fused gradient average +
// momentum update.  All reductions run in a fixed order, so results
// are identical from run to run.
#include <algorithm>

#include "device_common.h"
#include "internal.h"
#include "prep.h"

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

// ---- layout conversions --------------------------------------------------------------------

__device__ __forceinline__ unsigned fdivu(const FastDiv& f, unsigned n)
{
    return (__umulhi(n, f.m) + n) >> f.s;
}

// dst[n][hw][c] = x[n][c][hw]: one thread per (n, hw) position, channels in a loop, so that
// the reads (consecutive hw per channel plane) and the writes (consecutive positions) both
// coalesce.
template <typename T>
__global__ __launch_bounds__(256) void to_nhwc_kernel(const float* __restrict__ x,
                                                      T* __restrict__ dst, int positions, int C,
                                                      int HW, FastDiv fhw)
{
    const int t = blockIdx.x * 256 + threadIdx.x;
    if (t >= positions) return;
    const unsigned n = fdivu(fhw, (unsigned)t), hw = (unsigned)t - n * (unsigned)HW;
    const float* src = x + (long long)n * C * HW + hw;
    T* out = dst + (long long)t * C;
    for (int c = 0; c < C; ++c) out[c] = from_f32<T>(src[(long long)c * HW]);
}

hipError_t to_nhwc(Dt dt, const float* x, void* dst, int N, int C, int HW, hipStream_t s)
{
    const long long positions = (long long)N * HW;
    if (positions <= 0 || C <= 0) return hipSuccess;
    const FastDiv fhw = make_fastdiv((unsigned)HW);
    dim3 g(grid_for((size_t)positions, 256));
    if (dt == DT_F32)
        hipLaunchKernelGGL(to_nhwc_kernel<float>, g, dim3(256), 0, s, x, static_cast<float*>(dst),
                           (int)positions, C, HW, fhw);
    else
        hipLaunchKernelGGL(to_nhwc_kernel<bf16_t>, g, dim3(256), 0, s, x,
                           static_cast<bf16_t*>(dst), (int)positions, C, HW, fhw);
    return hipGetLastError();
}

// X'[n][PD + h][PD + w][c] = x[n][c][h][w] for c < C: one thread per pixel, channels in a loop.
// CP > 0 (= Cp, 8 or 16 bytes of channels): the pixel's channels, zeros included, go out as one
// vector store, so every byte of the written lines is written.
template <typename T, int CP>
__global__ __launch_bounds__(256) void to_nhwc_padded_kernel(const float* __restrict__ x,
                                                             T* __restrict__ dst, int pixels,
                                                             int C, int H, int W, int PD,
                                                             int Hp, int Wp, int Cp, FastDiv fw,
                                                             FastDiv fh)
{
    const int t = blockIdx.x * 256 + threadIdx.x;
    if (t >= pixels) return;
    const unsigned r = fdivu(fw, (unsigned)t), w = (unsigned)t - r * (unsigned)W;
    const unsigned n = fdivu(fh, r), h = r - n * (unsigned)H;
    const float* src = x + ((long long)n * C * H + h) * W + w;
    T* out = dst + (((long long)n * Hp + PD + h) * Wp + PD + w) * Cp;
    if constexpr (CP > 0) {
        static_assert(CP * sizeof(T) == 8 || CP * sizeof(T) == 16, "vector width");
        T v[CP];
#pragma unroll
        for (int c = 0; c < CP; ++c) v[c] = from_f32<T>(c < C ? src[(long long)c * H * W] : 0.f);
        if constexpr (CP * sizeof(T) == 16) *reinterpret_cast<uint4*>(out) = *reinterpret_cast<const uint4*>(v);
        else *reinterpret_cast<uint2*>(out) = *reinterpret_cast<const uint2*>(v);
    } else {
        for (int c = 0; c < C; ++c) out[c] = from_f32<T>(src[(long long)c * H * W]);
    }
}

hipError_t to_nhwc_padded(Dt dt, const float* x, void* dst, int N, int C, int H, int W,
                          int PD, const RunGeom& r, hipStream_t s)
{
    const long long pixels = (long long)N * H * W;
    if (pixels <= 0 || C <= 0) return hipSuccess;
    const FastDiv fw = make_fastdiv((unsigned)W), fh = make_fastdiv((unsigned)H);
    dim3 g(grid_for((size_t)pixels, 256));
    if (dt == DT_F32) {
        float* o = static_cast<float*>(dst);
        if (r.Cp == 2)
            hipLaunchKernelGGL((to_nhwc_padded_kernel<float, 2>), g, dim3(256), 0, s, x, o,
                               (int)pixels, C, H, W, PD, r.Hp, r.Wp, r.Cp, fw, fh);
        else if (r.Cp == 4)
            hipLaunchKernelGGL((to_nhwc_padded_kernel<float, 4>), g, dim3(256), 0, s, x, o,
                               (int)pixels, C, H, W, PD, r.Hp, r.Wp, r.Cp, fw, fh);
        else
            hipLaunchKernelGGL((to_nhwc_padded_kernel<float, 0>), g, dim3(256), 0, s, x, o,
                               (int)pixels, C, H, W, PD, r.Hp, r.Wp, r.Cp, fw, fh);
    } else {
        bf16_t* o = static_cast<bf16_t*>(dst);
        if (r.Cp == 4)
            hipLaunchKernelGGL((to_nhwc_padded_kernel<bf16_t, 4>), g, dim3(256), 0, s, x, o,
                               (int)pixels, C, H, W, PD, r.Hp, r.Wp, r.Cp, fw, fh);
        else if (r.Cp == 8)
            hipLaunchKernelGGL((to_nhwc_padded_kernel<bf16_t, 8>), g, dim3(256), 0, s, x, o,
                               (int)pixels, C, H, W, PD, r.Hp, r.Wp, r.Cp, fw, fh);
        else
            hipLaunchKernelGGL((to_nhwc_padded_kernel<bf16_t, 0>), g, dim3(256), 0, s, x, o,
                               (int)pixels, C, H, W, PD, r.Hp, r.Wp, r.Cp, fw, fh);
    }
    return hipGetLastError();
}

// ---- weight preparation ---------------------------------------------------------------------
// One launch serves every job; job j owns blocks [block0_j, block0_{j+1}) and each block
// converts kPrepPerBlock consecutive destination elements.  The source index of a destination
// element follows from its layout (see PrepKind).

int prep_blocks(int n) { return (n + kPrepPerBlock - 1) / kPrepPerBlock; }

void prep_fill_divisors(PrepJob& j)
{
    switch (j.kind) {
    case PREP_CONV_F:
        j.f0 = make_fastdiv((unsigned)(j.KK * j.cg));
        j.f1 = make_fastdiv((unsigned)j.cg);
        break;
    case PREP_CONV_D:
        j.f0 = make_fastdiv((unsigned)j.og);
        j.f1 = make_fastdiv((unsigned)j.KK);
        j.f2 = make_fastdiv((unsigned)j.cg);
        break;
    case PREP_CONV_C:
        j.f0 = make_fastdiv((unsigned)j.og);
        j.f1 = make_fastdiv((unsigned)j.cg);
        j.f2 = make_fastdiv((unsigned)j.KK);
        break;
    case PREP_FC_PERM:
        j.f0 = make_fastdiv((unsigned)j.IN);
        j.f1 = make_fastdiv((unsigned)j.C);
        break;
    case PREP_CONV_RUN:
        j.f0 = make_fastdiv((unsigned)j.RUN);
        j.f1 = make_fastdiv((unsigned)j.Cp);
        break;
    default:
        break;
    }
}

template <typename T>
__global__ __launch_bounds__(256) void prep_kernel(const PrepJob* __restrict__ jobs, int njobs,
                                                   const float* __restrict__ w,
                                                   T* __restrict__ dst)
{
    prep_block<T>(jobs, njobs, w, dst, (int)blockIdx.x);
}

hipError_t prep_weights(Dt dt, const PrepJob* jobs, int njobs, int blocks, const float* w,
                        void* dst, hipStream_t s)
{
    if (njobs <= 0 || blocks <= 0) return hipSuccess;
    if (dt == DT_F32)
        hipLaunchKernelGGL(prep_kernel<float>, dim3(blocks), dim3(256), 0, s, jobs, njobs, w,
                           static_cast<float*>(dst));
    else
        hipLaunchKernelGGL(prep_kernel<bf16_t>, dim3(blocks), dim3(256), 0, s, jobs, njobs, w,
                           static_cast<bf16_t*>(dst));
    return hipGetLastError();
}

// ---- max-pooling over NHWC tensors ------------------------------------------------------------
// KT / ST > 0: window and stride known at compile time (2/2 and 3/2 are the common cases).
// CV channels per thread (16 bytes of channels when C allows it, else 1).  A pooled tensor that
// feeds a fully connected layer is stored NCHW instead (the (c, h, w) order that layer reads);
// argmax always follows the layout of the pooled tensor.

template <typename T, int CV> struct Chans {
    T v[CV];
};

template <typename T, int CV>
__device__ __forceinline__ Chans<T, CV> load_chans(const T* p)
{
    Chans<T, CV> r;
    if constexpr (CV * sizeof(T) == 16) {
        *reinterpret_cast<uint4*>(r.v) = *reinterpret_cast<const uint4*>(p);
    } else {
#pragma unroll
        for (int i = 0; i < CV; ++i) r.v[i] = p[i];
    }
    return r;
}

template <typename T, int CV>
__device__ __forceinline__ void store_chans(T* p, const Chans<T, CV>& r)
{
    if constexpr (CV * sizeof(T) == 16) {
        *reinterpret_cast<uint4*>(p) = *reinterpret_cast<const uint4*>(r.v);
    } else {
#pragma unroll
        for (int i = 0; i < CV; ++i) p[i] = r.v[i];
    }
}

// One thread per CV channels of one output: the first maximal element of the K x K window in
// row-major window order; argmax holds its window position u*K + v.
template <typename T, int KT, int ST, int CV>
__global__ __launch_bounds__(256) void pool_fwd_kernel(int total, int C, int H, int W, int Kr,
                                                       int Sr, int OH, int OW, int out_nchw,
                                                       FastDiv fcv, FastDiv fow, FastDiv foh,
                                                       const T* __restrict__ x,
                                                       T* __restrict__ y,
                                                       uint8_t* __restrict__ argmax)
{
    const int K = KT > 0 ? KT : Kr, S = ST > 0 ? ST : Sr;
    // overlapping windows (S < K): blocks numbered so that each of the 8 XCDs (blocks go to them
    // round-robin) takes one contiguous range of outputs, and neighbouring output rows, which
    // read the same input rows, share that XCD's L2 (AlexNet's 3/2 poolings 50.6 / 32.9 ->
    // 47.8 / 31.2 us; disjoint 2/2 windows gain nothing from it)
    const unsigned nb = gridDim.x, hb = blockIdx.x, xq = nb / 8, xr = nb % 8, xx = hb % 8;
    const unsigned bid = S < K ? xx * xq + min(xx, xr) + hb / 8 : hb;
    const int t = (int)bid * 256 + threadIdx.x;  // over N*OH*OW*(C/CV)
    if (t >= total) return;
    const unsigned CG = (unsigned)(C / CV);
    const unsigned pos = fdivu(fcv, (unsigned)t), c0 = ((unsigned)t - pos * CG) * CV;
    const unsigned r = fdivu(fow, pos), j = pos - r * (unsigned)OW;
    const unsigned n = fdivu(foh, r), i = r - n * (unsigned)OH;
    const T* xp = x + (((int)n * H + (int)i * S) * W + (int)j * S) * C + (int)c0;
    const int rs = W * C;
    Chans<T, CV> best = load_chans<T, CV>(xp);
    float bv[CV];
    uint8_t bi[CV];
#pragma unroll
    for (int e = 0; e < CV; ++e) { bv[e] = to_f32<T>(best.v[e]); bi[e] = 0; }
    for (int u = 0; u < K; ++u)
        for (int v = 0; v < K; ++v) {
            const Chans<T, CV> cur = load_chans<T, CV>(xp + u * rs + v * C);
#pragma unroll
            for (int e = 0; e < CV; ++e) {
                const float tv = to_f32<T>(cur.v[e]);
                if (tv > bv[e]) { bv[e] = tv; best.v[e] = cur.v[e]; bi[e] = (uint8_t)(u * K + v); }
            }
        }
    if (out_nchw) {
#pragma unroll
        for (int e = 0; e < CV; ++e) {
            const int o = (((int)n * C + (int)c0 + e) * OH + (int)i) * OW + (int)j;
            y[o] = best.v[e];
            argmax[o] = bi[e];
        }
        return;
    }
    const int o = (int)pos * C + (int)c0;
    store_chans<T, CV>(y + o, best);
#pragma unroll
    for (int e = 0; e < CV; ++e) argmax[o + e] = bi[e];
}

// NCHW output (the pooled tensor feeds a fully connected layer): a block takes one sample and cb
// channels (a multiple of CV), computes their cb x P outputs (P = OH*OW; one task per position
// and CV channels, the same window rule as above) into LDS in the output's [channel][position]
// order, and writes them -- one contiguous range of y and one of argmax -- with 16-byte stores
// (one thread per position writing its CV channels to CV planes made 16 scattered narrow stores
// per thread: AlexNet pool3 ran at a third of the HBM rate).
constexpr int kPoolFwdCB = 64;              // channels per block at most
constexpr size_t kPoolFwdLds = 48 << 10;    // LDS bytes per block at most
template <typename T, int KT, int ST, int CV>
__global__ __launch_bounds__(256) void pool_fwd_nchw_kernel(int C, int H, int W, int Kr, int Sr,
                                                            int OH, int OW, int cb, FastDiv fcg,
                                                            const T* __restrict__ x,
                                                            T* __restrict__ y,
                                                            uint8_t* __restrict__ argmax)
{
    extern __shared__ __attribute__((aligned(16))) unsigned char pool_smem[];
    const int K = KT > 0 ? KT : Kr, S = ST > 0 ? ST : Sr;
    const int P = OH * OW, cgs = cb / CV;
    T* sy = reinterpret_cast<T*>(pool_smem);
    uint8_t* sa = pool_smem + (((size_t)cb * P * sizeof(T) + 15) & ~(size_t)15);
    const int n = blockIdx.y, cb0 = blockIdx.x * cb;
    for (int tk = threadIdx.x; tk < P * cgs; tk += 256) {
        const unsigned pos = fdivu(fcg, (unsigned)tk), cg = (unsigned)tk - pos * (unsigned)cgs;
        const unsigned i = pos / (unsigned)OW, j = pos - i * (unsigned)OW;
        const int c0 = cb0 + (int)cg * CV;
        const T* xp = x + (((long long)n * H + (int)i * S) * W + (int)j * S) * C + c0;
        const int rs = W * C;
        Chans<T, CV> best = load_chans<T, CV>(xp);
        float bv[CV];
        uint8_t bi[CV];
#pragma unroll
        for (int e = 0; e < CV; ++e) { bv[e] = to_f32<T>(best.v[e]); bi[e] = 0; }
        for (int u = 0; u < K; ++u)
            for (int v = 0; v < K; ++v) {
                const Chans<T, CV> cur = load_chans<T, CV>(xp + u * rs + v * C);
#pragma unroll
                for (int e = 0; e < CV; ++e) {
                    const float tv = to_f32<T>(cur.v[e]);
                    if (tv > bv[e]) { bv[e] = tv; best.v[e] = cur.v[e]; bi[e] = (uint8_t)(u * K + v); }
                }
            }
#pragma unroll
        for (int e = 0; e < CV; ++e) {
            sy[((int)cg * CV + e) * P + (int)pos] = best.v[e];
            sa[((int)cg * CV + e) * P + (int)pos] = bi[e];
        }
    }
    __syncthreads();
    const long long base = ((long long)n * C + cb0) * P;
    const int cnt = cb * P;
    T* yo = y + base;
    uint8_t* ao = argmax + base;
    constexpr int VE = 16 / (int)sizeof(T);
    if (base % VE == 0 && cnt % VE == 0)
        for (int e = threadIdx.x; e < cnt / VE; e += 256)
            *reinterpret_cast<uint4*>(yo + (long long)e * VE) = *reinterpret_cast<const uint4*>(sy + e * VE);
    else
        for (int e = threadIdx.x; e < cnt; e += 256) yo[e] = sy[e];
    if (base % 16 == 0 && cnt % 16 == 0)
        for (int e = threadIdx.x; e < cnt / 16; e += 256)
            *reinterpret_cast<uint4*>(ao + (long long)e * 16) = *reinterpret_cast<const uint4*>(sa + e * 16);
    else
        for (int e = threadIdx.x; e < cnt; e += 256) ao[e] = sa[e];
}

template <typename T, int CV>
static void pool_fwd_launch(int N, int C, int H, int W, int K, int S, bool out_nchw,
                            const void* x, void* y, uint8_t* argmax, hipStream_t s)
{
    const int OH = (H - K) / S + 1, OW = (W - K) / S + 1;
    if (out_nchw && CV > 1) {
        // channels per block: the largest multiple of CV dividing C within the limits
        const size_t P = (size_t)OH * OW;
        int cb = 0;
        for (int c = std::min(kPoolFwdCB, C); c >= CV && !cb; --c)
            if (C % c == 0 && c % CV == 0 &&
                (((size_t)c * P * sizeof(T) + 15) & ~(size_t)15) + (size_t)c * P <= kPoolFwdLds)
                cb = c;
        if (cb > 0) {
            const size_t shm = (((size_t)cb * P * sizeof(T) + 15) & ~(size_t)15) + (size_t)cb * P;
            const dim3 g((unsigned)(C / cb), (unsigned)N);
            const FastDiv fcg = make_fastdiv((unsigned)(cb / CV));
            const T* xx = static_cast<const T*>(x);
            T* yy = static_cast<T*>(y);
            if (K == 3 && S == 2)
                hipLaunchKernelGGL((pool_fwd_nchw_kernel<T, 3, 2, CV>), g, dim3(256), shm, s, C, H,
                                   W, K, S, OH, OW, cb, fcg, xx, yy, argmax);
            else
                hipLaunchKernelGGL((pool_fwd_nchw_kernel<T, 0, 0, CV>), g, dim3(256), shm, s, C, H,
                                   W, K, S, OH, OW, cb, fcg, xx, yy, argmax);
            return;
        }
    }
    const int total = N * OH * OW * (C / CV);
    const FastDiv fcv = make_fastdiv((unsigned)(C / CV)), fow = make_fastdiv((unsigned)OW),
                  foh = make_fastdiv((unsigned)OH);
    dim3 g(grid_for(total, 256)), b(256);
    const T* xx = static_cast<const T*>(x);
    T* yy = static_cast<T*>(y);
    if (K == 2 && S == 2)
        hipLaunchKernelGGL((pool_fwd_kernel<T, 2, 2, CV>), g, b, 0, s, total, C, H, W, K, S, OH,
                           OW, (int)out_nchw, fcv, fow, foh, xx, yy, argmax);
    else if (K == 3 && S == 2)
        hipLaunchKernelGGL((pool_fwd_kernel<T, 3, 2, CV>), g, b, 0, s, total, C, H, W, K, S, OH,
                           OW, (int)out_nchw, fcv, fow, foh, xx, yy, argmax);
    else
        hipLaunchKernelGGL((pool_fwd_kernel<T, 0, 0, CV>), g, b, 0, s, total, C, H, W, K, S, OH,
                           OW, (int)out_nchw, fcv, fow, foh, xx, yy, argmax);
}

hipError_t pool_fwd(Dt dt, int N, int C, int H, int W, int K, int S, bool out_nchw,
                    const void* x, void* y, uint8_t* argmax, hipStream_t s)
{
    const int OH = (H - K) / S + 1, OW = (W - K) / S + 1;
    if ((long long)N * C * OH * OW <= 0) return hipSuccess;
    if (dt == DT_F32) {
        if (C % 4 == 0) pool_fwd_launch<float, 4>(N, C, H, W, K, S, out_nchw, x, y, argmax, s);
        else pool_fwd_launch<float, 1>(N, C, H, W, K, S, out_nchw, x, y, argmax, s);
    } else {
        if (C % 8 == 0) pool_fwd_launch<bf16_t, 8>(N, C, H, W, K, S, out_nchw, x, y, argmax, s);
        else pool_fwd_launch<bf16_t, 1>(N, C, H, W, K, S, out_nchw, x, y, argmax, s);
    }
    return hipGetLastError();
}

// The ReLU mask of the layer that produced a pooled tensor, as seen by the pooling backward:
// a window's output gradient goes to the position of its maximum, and the value there is the
// window's pooled output, so a window whose pooled output is not positive contributes nothing.
// The gate is that pooled output (same index as the output gradient), or null without ReLU.
template <typename T>
__device__ __forceinline__ bool gate_open(const T* gate, long long o)
{
    return !gate || to_f32<T>(gate[o]) > 0.f;
}

// Input gradient of a pooling, general window and stride, NHWC (the output gradient NCHW when
// dy_nchw is set): one thread per CV channels of one input element, the sum in ascending window
// order of the output gradients of the windows whose maximum sits there (windows overlap when
// S < K); gathering keeps it free of atomics.
template <typename T, int CV>
__global__ __launch_bounds__(256) void pool_bwd_kernel(int total, int C, int H, int W, int K,
                                                       int S, int OH, int OW, int dy_nchw,
                                                       FastDiv fcv,
                                                       FastDiv fw, FastDiv fh,
                                                       const uint8_t* __restrict__ argmax,
                                                       const T* __restrict__ dy,
                                                       const T* __restrict__ gate,
                                                       T* __restrict__ dx)
{
    const int t = blockIdx.x * 256 + threadIdx.x;  // over N*H*W*(C/CV)
    if (t >= total) return;
    const unsigned CG = (unsigned)(C / CV);
    const unsigned pos = fdivu(fcv, (unsigned)t), c0 = ((unsigned)t - pos * CG) * CV;
    const unsigned r = fdivu(fw, pos), wu = pos - r * (unsigned)W;
    const unsigned n = fdivu(fh, r), hu = r - n * (unsigned)H;
    const int h = (int)hu, w = (int)wu;
    float acc[CV];
#pragma unroll
    for (int e = 0; e < CV; ++e) acc[e] = 0.f;
    // windows i with i*S <= h <= i*S + K - 1
    const int ilo = h - K + 1 <= 0 ? 0 : (h - K + 1 + S - 1) / S;
    const int ihi = min(h / S, OH - 1);
    const int jlo = w - K + 1 <= 0 ? 0 : (w - K + 1 + S - 1) / S;
    const int jhi = min(w / S, OW - 1);
    for (int i = ilo; i <= ihi; ++i)
        for (int j = jlo; j <= jhi; ++j) {
            const uint8_t here = (uint8_t)((h - i * S) * K + (w - j * S));
#pragma unroll
            for (int e = 0; e < CV; ++e) {
                const int o = dy_nchw ? (((int)n * C + (int)c0 + e) * OH + i) * OW + j
                                      : (((int)n * OH + i) * OW + j) * C + (int)c0 + e;
                if (argmax[o] == here && gate_open(gate, o)) acc[e] += to_f32<T>(dy[o]);
            }
        }
    Chans<T, CV> out;
#pragma unroll
    for (int e = 0; e < CV; ++e) out.v[e] = from_f32<T>(acc[e]);
    store_chans<T, CV>(dx + (int)pos * C + (int)c0, out);
}

// The same for stride 2 and a 2 x 2 or 3 x 3 window, NHWC: one thread per CV channels of a
// 2 x 2 block of input positions.  The windows touching the block (one for K = 2, up to four
// for K = 3) are read once and each routes its output gradient to the block position that holds
// its maximum; every position adds its windows in ascending (i, j) order, as above.
template <typename T, int K, int CV>
__global__ __launch_bounds__(256) void pool_bwd_s2_kernel(int total, int C, int H, int W, int OH,
                                                          int OW, int BH, int BW, FastDiv fcv,
                                                          FastDiv fbw, FastDiv fbh,
                                                          const uint8_t* __restrict__ argmax,
                                                          const T* __restrict__ dy,
                                                          const T* __restrict__ gate,
                                                          T* __restrict__ dx)
{
    static_assert(K == 2 || K == 3, "window");
    const int t = blockIdx.x * 256 + threadIdx.x;  // over N*BH*BW*(C/CV)
    if (t >= total) return;
    const unsigned CG = (unsigned)(C / CV);
    const unsigned pos = fdivu(fcv, (unsigned)t), c0 = ((unsigned)t - pos * CG) * CV;
    const unsigned r = fdivu(fbw, pos), bw = pos - r * (unsigned)BW;
    const unsigned n = fdivu(fbh, r), bh = r - n * (unsigned)BH;
    float acc[2][2][CV];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int e = 0; e < CV; ++e) acc[a][b][e] = 0.f;
#pragma unroll
    for (int di = 0; di < K - 1; ++di) {
        const int i = (int)bh - (K - 2) + di;  // window row; block row 2*bh sits at u = 2*(bh-i)
        if (i < 0 || i >= OH) continue;
#pragma unroll
        for (int dj = 0; dj < K - 1; ++dj) {
            const int j = (int)bw - (K - 2) + dj;
            if (j < 0 || j >= OW) continue;
            const int o = (((int)n * OH + i) * OW + j) * C + (int)c0;
            const Chans<T, CV> g = load_chans<T, CV>(dy + o);
            uint8_t am[CV];
            if constexpr (CV == 8) *reinterpret_cast<uint2*>(am) = *reinterpret_cast<const uint2*>(argmax + o);
            else if constexpr (CV == 4) *reinterpret_cast<unsigned*>(am) = *reinterpret_cast<const unsigned*>(argmax + o);
            else am[0] = argmax[o];
            float gv[CV];
#pragma unroll
            for (int e = 0; e < CV; ++e) gv[e] = to_f32<T>(g.v[e]);
            if (gate) {
                const Chans<T, CV> y = load_chans<T, CV>(gate + o);
#pragma unroll
                for (int e = 0; e < CV; ++e)
                    if (!(to_f32<T>(y.v[e]) > 0.f)) gv[e] = 0.f;
            }
#pragma unroll
            for (int dh = 0; dh < 2; ++dh) {
                const int u = dh + 2 * (K - 2) - 2 * di;
                if (u < 0 || u >= K) continue;
#pragma unroll
                for (int dw = 0; dw < 2; ++dw) {
                    const int v = dw + 2 * (K - 2) - 2 * dj;
                    if (v < 0 || v >= K) continue;
#pragma unroll
                    for (int e = 0; e < CV; ++e)
                        if (am[e] == u * K + v) acc[dh][dw][e] += gv[e];
                }
            }
        }
    }
    const int h0 = 2 * (int)bh, w0 = 2 * (int)bw;
#pragma unroll
    for (int dh = 0; dh < 2; ++dh)
#pragma unroll
        for (int dw = 0; dw < 2; ++dw) {
            if (h0 + dh >= H || w0 + dw >= W) continue;
            Chans<T, CV> out;
#pragma unroll
            for (int e = 0; e < CV; ++e) out.v[e] = from_f32<T>(acc[dh][dw][e]);
            store_chans<T, CV>(dx + (((int)n * H + h0 + dh) * W + w0 + dw) * C + (int)c0, out);
        }
}

// Pooling backward whose output gradient is NCHW (the pooled tensor feeds a fully connected
// layer) and whose input gradient is NHWC.  A block takes one sample, cb channels and a band of
// input rows: it reads the output gradients (gated) and window maxima of the windows over that
// band, contiguous per channel, into LDS (channel rows padded to an odd length), then one thread
// per (position, channel), channels fastest, gathers in ascending window order and writes NHWC.
constexpr int kPoolCB = 64;            // channels per block at most
constexpr size_t kPoolLds = 64 << 10;  // LDS bytes per block at most
template <typename T, int KT, int ST, int CV>
__global__ __launch_bounds__(256) void pool_bwd_nchw_kernel(int C, int H, int W, int Kr, int Sr,
                                                            int OH, int OW, int cb, int pst,
                                                            int rows, FastDiv fcb, FastDiv fw,
                                                            FastDiv fs,
                                                            const uint8_t* __restrict__ argmax,
                                                            const T* __restrict__ dy,
                                                            const T* __restrict__ gate,
                                                            T* __restrict__ dx)
{
    const int K = KT > 0 ? KT : Kr, S = ST > 0 ? ST : Sr;
    extern __shared__ float sg[];  // [cb][pst] gradients, then [cb][pst] maxima
    uint8_t* sa = reinterpret_cast<uint8_t*>(sg + cb * pst);
    const int n = blockIdx.y, cb0 = blockIdx.x * cb;
    const int h0 = blockIdx.z * rows, h1 = min(H, h0 + rows);
    if (h0 >= H) return;
    // windows over rows [h0, h1): i in [ilo, ihi]
    const int ilo = h0 - K + 1 <= 0 ? 0 : (h0 - K + 1 + S - 1) / S;
    const int ihi = min((h1 - 1) / S, OH - 1);
    const int nwin = (ihi - ilo + 1) * OW;
    const long long base = ((long long)n * C + cb0) * OH * OW + (long long)ilo * OW;
    for (int e = threadIdx.x; e < cb * nwin; e += 256) {
        const int cl = e / nwin, ij = e - cl * nwin;
        const long long g = base + (long long)cl * OH * OW + ij;
        sg[cl * pst + ij] = gate_open(gate, g) ? to_f32<T>(dy[g]) : 0.f;
        sa[cl * pst + ij] = argmax[g];
    }
    __syncthreads();
    // one thread per (position, CV channels), channel groups fastest; CV = 8 (bf16) or 4 (fp32)
    // channels go out as one 16-byte store (one 2-byte store per thread made the store
    // instructions, not the bytes, the limit: 75 us for the 67 MB input gradient of the
    // bottleneck network's 4/4 pooling)
    const int cbv = cb / CV;  // fcb divides by cbv
    const int cnt = (h1 - h0) * W * cbv;
    // (the window ranges divide non-negative values by the stride: by a constant, or with the
    // fast division by an invariant integer)
    auto divs = [&](int v) { return ST > 0 ? v / ST : (int)fdivu(fs, (unsigned)v); };
    for (int e = threadIdx.x; e < cnt; e += 256) {
        const unsigned hw = fdivu(fcb, (unsigned)e), cg = (unsigned)e - hw * (unsigned)cbv;
        const unsigned hr = fdivu(fw, hw);
        const int h = h0 + (int)hr, w = (int)(hw - hr * (unsigned)W);
        const int jlo = w - K + 1 <= 0 ? 0 : divs(w - K + 1 + S - 1);
        const int jhi = min(divs(w), OW - 1);
        const int il = max(ilo, h - K + 1 <= 0 ? 0 : divs(h - K + 1 + S - 1));
        const int ih = min(divs(h), OH - 1);
        const int cl0 = (int)cg * CV;
        float acc[CV];
#pragma unroll
        for (int k = 0; k < CV; ++k) acc[k] = 0.f;
        for (int i = il; i <= ih; ++i)
            for (int j = jlo; j <= jhi; ++j) {
                const int wi = (i - ilo) * OW + j;
                const uint8_t code = (uint8_t)((h - i * S) * K + (w - j * S));
#pragma unroll
                for (int k = 0; k < CV; ++k) {
                    const int idx = (cl0 + k) * pst + wi;
                    if (sa[idx] == code) acc[k] += sg[idx];
                }
            }
        Chans<T, CV> out;
#pragma unroll
        for (int k = 0; k < CV; ++k) out.v[k] = from_f32<T>(acc[k]);
        store_chans<T, CV>(dx + (((long long)n * H + h) * W + w) * C + cb0 + cl0, out);
    }
}

template <typename T, int CV>
static void pool_bwd_launch(int N, int C, int H, int W, int K, int S, bool dy_nchw,
                            const uint8_t* argmax, const void* dy, void* dx, const void* gate,
                            hipStream_t s)
{
    const int OH = (H - K) / S + 1, OW = (W - K) / S + 1;
    const T* d = static_cast<const T*>(dy);
    const T* gt = static_cast<const T*>(gate);
    T* o = static_cast<T*>(dx);
    dim3 b(256);
    if (dy_nchw) {
        // channels per block: the largest divisor of C within the limits; row bands so that
        // the launch has at least about 2048 blocks
        const int pst = (OH * OW) | 1;
        const int cmax = (int)std::min<size_t>(kPoolCB, kPoolLds / ((size_t)pst * (sizeof(float) + 1)));
        int cb = 0;
        for (int c = std::min(cmax, C); c >= 1 && !cb; --c)
            if (C % c == 0) cb = c;
        if (cb > 0) {
            const long long pairs = (long long)N * (C / cb);
            const int bands = (int)std::max(1ll, std::min<long long>(H, (2048 + pairs - 1) / pairs));
            const int rows = (H + bands - 1) / bands;
            const size_t shm = (size_t)cb * pst * (sizeof(float) + 1);
            dim3 g((unsigned)(C / cb), (unsigned)N, (unsigned)((H + rows - 1) / rows));
            const FastDiv fw = make_fastdiv((unsigned)W), fs = make_fastdiv((unsigned)S);
            constexpr int V = 16 / sizeof(T);
            if (cb % V == 0) {
                const FastDiv fcb = make_fastdiv((unsigned)(cb / V));
                if (K == 2 && S == 2)
                    hipLaunchKernelGGL((pool_bwd_nchw_kernel<T, 2, 2, V>), g, b, shm, s, C, H, W,
                                       K, S, OH, OW, cb, pst, rows, fcb, fw, fs, argmax, d, gt, o);
                else if (K == 3 && S == 2)
                    hipLaunchKernelGGL((pool_bwd_nchw_kernel<T, 3, 2, V>), g, b, shm, s, C, H, W,
                                       K, S, OH, OW, cb, pst, rows, fcb, fw, fs, argmax, d, gt, o);
                else if (K == 4 && S == 4)
                    hipLaunchKernelGGL((pool_bwd_nchw_kernel<T, 4, 4, V>), g, b, shm, s, C, H, W,
                                       K, S, OH, OW, cb, pst, rows, fcb, fw, fs, argmax, d, gt, o);
                else
                    hipLaunchKernelGGL((pool_bwd_nchw_kernel<T, 0, 0, V>), g, b, shm, s, C, H, W,
                                       K, S, OH, OW, cb, pst, rows, fcb, fw, fs, argmax, d, gt, o);
            } else {
                const FastDiv fcb = make_fastdiv((unsigned)cb);
                hipLaunchKernelGGL((pool_bwd_nchw_kernel<T, 0, 0, 1>), g, b, shm, s, C, H, W, K,
                                   S, OH, OW, cb, pst, rows, fcb, fw, fs, argmax, d, gt, o);
            }
            return;
        }
    }
    const FastDiv fcv = make_fastdiv((unsigned)(C / CV));
    if (!dy_nchw && S == 2 && (K == 2 || K == 3)) {
        const int BH = (H + 1) / 2, BW = (W + 1) / 2;
        const int total = N * BH * BW * (C / CV);
        const FastDiv fbw = make_fastdiv((unsigned)BW), fbh = make_fastdiv((unsigned)BH);
        dim3 g(grid_for(total, 256));
        if (K == 2)
            hipLaunchKernelGGL((pool_bwd_s2_kernel<T, 2, CV>), g, b, 0, s, total, C, H, W, OH,
                               OW, BH, BW, fcv, fbw, fbh, argmax, d, gt, o);
        else
            hipLaunchKernelGGL((pool_bwd_s2_kernel<T, 3, CV>), g, b, 0, s, total, C, H, W, OH,
                               OW, BH, BW, fcv, fbw, fbh, argmax, d, gt, o);
        return;
    }
    const int total = N * H * W * (C / CV);
    const FastDiv fw = make_fastdiv((unsigned)W), fh = make_fastdiv((unsigned)H);
    hipLaunchKernelGGL((pool_bwd_kernel<T, CV>), dim3(grid_for(total, 256)), b, 0, s, total, C,
                       H, W, K, S, OH, OW, (int)dy_nchw, fcv, fw, fh, argmax, d, gt, o);
}

hipError_t pool_bwd(Dt dt, int N, int C, int H, int W, int K, int S, bool dy_nchw,
                    const uint8_t* argmax, const void* dy, void* dx, const void* gate,
                    hipStream_t s)
{
    if ((long long)N * C * H * W <= 0) return hipSuccess;
    if (dt == DT_F32) {
        if (C % 4 == 0) pool_bwd_launch<float, 4>(N, C, H, W, K, S, dy_nchw, argmax, dy, dx, gate, s);
        else pool_bwd_launch<float, 1>(N, C, H, W, K, S, dy_nchw, argmax, dy, dx, gate, s);
    } else {
        if (C % 8 == 0) pool_bwd_launch<bf16_t, 8>(N, C, H, W, K, S, dy_nchw, argmax, dy, dx, gate, s);
        else pool_bwd_launch<bf16_t, 1>(N, C, H, W, K, S, dy_nchw, argmax, dy, dx, gate, s);
    }
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
// compute type.  With loss_out set, the batch-mean loss is formed in the same launch: every
// block writes the sum of its four rows, and the block that finishes last adds those block sums
// in block order (a counter in `sync` elects it and is reset by it), so the value does not
// depend on the order in which blocks run.
template <typename T>
__global__ __launch_bounds__(256) void softmax_xent_kernel(int B, int NC, float inv_nb,
                                                           const float* __restrict__ z,
                                                           const int32_t* __restrict__ labels,
                                                           T* __restrict__ dz,
                                                           float* __restrict__ block_sums,
                                                           unsigned* __restrict__ sync,
                                                           float* __restrict__ loss_out)
{
    __shared__ float rows[4];
    __shared__ bool last;
    const int wave = threadIdx.x >> 6;
    const int row = blockIdx.x * 4 + wave;
    const int lane = threadIdx.x & 63;
    float loss = 0.f;
    if (row < B) {
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
        loss = valid ? lse - zr[y] : __int_as_float(0x7fc00000);
    }
    if (!loss_out) return;
    if (lane == 0) rows[wave] = loss;
    __syncthreads();
    if (threadIdx.x == 0) {
        __hip_atomic_store(&block_sums[blockIdx.x], ((rows[0] + rows[1]) + rows[2]) + rows[3],
                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __threadfence();
        last = atomicAdd(sync, 1u) == gridDim.x - 1;
    }
    __syncthreads();
    if (!last) return;
    // the last block: every thread fetches block sums k = tid, tid+256, ... and adds them in
    // that order; thread 0 then adds the 256 results in thread order.
    __shared__ float part[256];
    __threadfence();
    float acc = 0.f;
    for (unsigned k = threadIdx.x; k < gridDim.x; k += 256)
        acc += __hip_atomic_load(&block_sums[k], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    part[threadIdx.x] = acc;
    __syncthreads();
    if (threadIdx.x == 0) {
        float tot = 0.f;
        for (int k = 0; k < 256; ++k) tot += part[k];
        loss_out[0] = tot / (float)B;
        *sync = 0u;
    }
}

hipError_t softmax_xent(Dt dt, int B, int NC, int Nb, const float* logits,
                        const int32_t* labels, void* dz, float* block_sums, unsigned* sync,
                        float* loss_out, hipStream_t s)
{
    const float inv = 1.0f / (float)Nb;
    dim3 grid((B + 3) / 4);
    if (dt == DT_F32)
        hipLaunchKernelGGL(softmax_xent_kernel<float>, grid, dim3(256), 0, s, B, NC, inv, logits,
                           labels, static_cast<float*>(dz), block_sums, sync, loss_out);
    else
        hipLaunchKernelGGL(softmax_xent_kernel<bf16_t>, grid, dim3(256), 0, s, B, NC, inv,
                           logits, labels, static_cast<bf16_t*>(dz), block_sums, sync, loss_out);
    return hipGetLastError();
}

// ---- gradient average + momentum update --------------------------------------------------------
//
// g = (1/R) sum_r grads[r][i] (ascending r, fp32), then v = mu*v + g and w = w - lr*v (each one
// fused multiply-add, i.e. one rounding), or w = w - lr*g without momentum.  Four consecutive
// elements per thread with 16-byte loads when every row is 16-byte aligned; the R loads of a
// thread are independent and issued before the adds.

typedef float f32x4 __attribute__((ext_vector_type(4)));

// The non-finite check of a step: an average-only pass sets *nonfinite when any average is not
// finite; the update pass that follows does nothing while *skip is set.  Both null otherwise.
struct FiniteGuard {
    const int* skip;
    int* nonfinite;
};

template <bool MOM, bool AVG, bool UPD>
__device__ __forceinline__ void avg_update_one(const float* __restrict__ grads, int R, long long ld,
                                               long long i, float* __restrict__ w,
                                               float* __restrict__ v, float lr, float mu,
                                               float* __restrict__ avg, int* nonfinite)
{
    float s = grads[i];
    for (int r = 1; r < R; ++r) s += grads[(long long)r * ld + i];
    float g = s / (float)R;
    if (AVG) avg[i] = g;
    if (AVG && !UPD && nonfinite && !__builtin_isfinite(g)) *nonfinite = 1;
    if (UPD) {
        if (MOM) {
            const float vn = fmaf(mu, v[i], g);
            v[i] = vn;
            g = vn;
        }
        w[i] = fmaf(-lr, g, w[i]);
    }
}

// n elements in 16-byte vectors: a block walks spans of 2 x 256 vectors (each thread two, 4 KB
// apart, so that every wave reads 1 KB contiguous per row and pass), issues the loads of w and v
// and then the rows, adding each row as it arrives in ascending r (the compiler keeps the loads
// in flight and waits for them one by one; holding all R rows in registers first took 166
// registers at R = 16 and three waves per SIMD instead of five: 5.48 against 5.97 TB/s); the
// n % 4 elements left over are taken by the first thread of the grid.  Every access is
// nontemporal (each byte is read or written once per call): measured at R = 16, n = 61M,
// 5.97 TB/s against 5.43 TB/s for one vector per thread with cached w and v.
template <int RT, bool MOM, bool AVG, bool UPD>
__global__ __launch_bounds__(256) void avg_update_vec4(const float* __restrict__ grads, int Rrt,
                                                       long long n, long long ld,
                                                       float* __restrict__ w,
                                                       float* __restrict__ v, float lr, float mu,
                                                       float* __restrict__ avg, FiniteGuard fg)
{
    if (UPD && fg.skip && *fg.skip) return;
    constexpr int U = 2;
    const long long n4 = n / 4, ld4 = ld / 4;
    const int R = RT > 0 ? RT : Rrt;
    const f32x4* g4 = reinterpret_cast<const f32x4*>(grads);
    f32x4* w4 = reinterpret_cast<f32x4*>(w);
    f32x4* v4 = reinterpret_cast<f32x4*>(v);
    for (long long base = (long long)blockIdx.x * 256 * U; base < n4;
         base += (long long)gridDim.x * 256 * U) {
        f32x4 s[U], wv[U], vv[U];
        bool ok[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const long long t = base + u * 256 + threadIdx.x;
            ok[u] = t < n4;
            s[u] = wv[u] = vv[u] = f32x4{0.f, 0.f, 0.f, 0.f};
            if (UPD && ok[u]) {
                wv[u] = __builtin_nontemporal_load(w4 + t);
                if (MOM) vv[u] = __builtin_nontemporal_load(v4 + t);
            }
        }
        if (RT > 0) {
#pragma unroll
            for (int r = 0; r < RT; ++r)
#pragma unroll
                for (int u = 0; u < U; ++u)
                    if (ok[u]) {
                        const f32x4 x = __builtin_nontemporal_load(g4 + r * ld4 + base +
                                                                   u * 256 + threadIdx.x);
                        s[u] = r == 0 ? x : s[u] + x;
                    }
        } else {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const long long t = base + u * 256 + threadIdx.x;
                if (!ok[u]) continue;
                s[u] = __builtin_nontemporal_load(g4 + t);
                for (int r = 1; r < R; ++r) s[u] += __builtin_nontemporal_load(g4 + r * ld4 + t);
            }
        }
        const float fr = (float)R;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const long long t = base + u * 256 + threadIdx.x;
            if (!ok[u]) continue;
            f32x4 g = {s[u][0] / fr, s[u][1] / fr, s[u][2] / fr, s[u][3] / fr};
            if (AVG) __builtin_nontemporal_store(g, reinterpret_cast<f32x4*>(avg) + t);
            if (AVG && !UPD && fg.nonfinite &&
                !(__builtin_isfinite(g[0]) && __builtin_isfinite(g[1]) && __builtin_isfinite(g[2]) &&
                  __builtin_isfinite(g[3])))
                *fg.nonfinite = 1;
            if (UPD) {
                if (MOM) {
#pragma unroll
                    for (int j = 0; j < 4; ++j) vv[u][j] = fmaf(mu, vv[u][j], g[j]);
                    __builtin_nontemporal_store(vv[u], v4 + t);
                    g = vv[u];
                }
#pragma unroll
                for (int j = 0; j < 4; ++j) wv[u][j] = fmaf(-lr, g[j], wv[u][j]);
                __builtin_nontemporal_store(wv[u], w4 + t);
            }
        }
    }
    if (blockIdx.x == 0 && threadIdx.x == 0)
        for (long long i = 4 * n4; i < n; ++i)
            avg_update_one<MOM, AVG, UPD>(grads, R, ld, i, w, v, lr, mu, avg, fg.nonfinite);
}

template <bool MOM, bool AVG, bool UPD>
__global__ __launch_bounds__(256) void avg_update_scalar(const float* __restrict__ grads, int R,
                                                         long long n, long long ld,
                                                         float* __restrict__ w,
                                                         float* __restrict__ v, float lr,
                                                         float mu, float* __restrict__ avg,
                                                         FiniteGuard fg)
{
    const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
    if (i >= n) return;
    if (UPD && fg.skip && *fg.skip) return;
    avg_update_one<MOM, AVG, UPD>(grads, R, ld, i, w, v, lr, mu, avg, fg.nonfinite);
}

// Dynamic LDS that the streaming average kernels reserve without using it, so that at most five
// 256-thread blocks share a compute unit (160 KB of LDS): fewer rows in flight at once keep the
// HBM row buffers open longer.  Measured (momentum kernel, blocks per CU unlimited / 4 / 5 / 6):
// R = 16, n = 61M 5.39 / 5.62 / 5.83 / 5.54 TB/s; R = 8, n = 61M 5.76 / 6.07 / 6.14 / 5.92;
// R = 16, n = 250M 5.44 / 5.53 / 5.69 / 5.57.  A launch with a capped grid (the layer-wise update
// beside other kernels) reserves nothing.
constexpr size_t kStreamLds = 160 * 1024 / 5 - 1024;

template <bool MOM, bool AVG, bool UPD>
static hipError_t avg_update_launch(const float* grads, int R, size_t n, size_t ld, float* w,
                                    float* v, float lr, float mu, float* avg, unsigned max_blocks,
                                    hipStream_t s, FiniteGuard fg)
{
    auto al = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; };
    const bool vec = (ld % 4 == 0) && al(grads) && (!AVG || al(avg)) && (!UPD || al(w)) &&
                     (!MOM || al(v));
    if (vec) {
        const long long nn = (long long)n;
        dim3 grid(grid_for(n / 4 + 1, 512));
        if (max_blocks && grid.x > max_blocks) grid.x = max_blocks;
        const size_t lds = max_blocks ? 0 : kStreamLds;
        switch (R) {
        case 1: hipLaunchKernelGGL((avg_update_vec4<1, MOM, AVG, UPD>), grid, dim3(256), lds, s, grads, R, nn, (long long)ld, w, v, lr, mu, avg, fg); break;
        case 2: hipLaunchKernelGGL((avg_update_vec4<2, MOM, AVG, UPD>), grid, dim3(256), lds, s, grads, R, nn, (long long)ld, w, v, lr, mu, avg, fg); break;
        case 4: hipLaunchKernelGGL((avg_update_vec4<4, MOM, AVG, UPD>), grid, dim3(256), lds, s, grads, R, nn, (long long)ld, w, v, lr, mu, avg, fg); break;
        case 8: hipLaunchKernelGGL((avg_update_vec4<8, MOM, AVG, UPD>), grid, dim3(256), lds, s, grads, R, nn, (long long)ld, w, v, lr, mu, avg, fg); break;
        case 16: hipLaunchKernelGGL((avg_update_vec4<16, MOM, AVG, UPD>), grid, dim3(256), lds, s, grads, R, nn, (long long)ld, w, v, lr, mu, avg, fg); break;
        default: hipLaunchKernelGGL((avg_update_vec4<0, MOM, AVG, UPD>), grid, dim3(256), lds, s, grads, R, nn, (long long)ld, w, v, lr, mu, avg, fg); break;
        }
    } else {
        hipLaunchKernelGGL((avg_update_scalar<MOM, AVG, UPD>), dim3(grid_for(n, 256)), dim3(256),
                           0, s, grads, R, (long long)n, (long long)ld, w, v, lr, mu, avg, fg);
    }
    return hipGetLastError();
}

hipError_t average_update(const float* grads, int R, size_t n, size_t ld, float* w, float* v,
                          float lr, float mu, float* avg, bool update, hipStream_t s,
                          unsigned max_blocks, const int* skip, int* nonfinite)
{
    const bool mom = update && mu != 0.0f;
    const bool wavg = avg != nullptr;
    const FiniteGuard fg{skip, nonfinite};
    if (!update) return avg_update_launch<false, true, false>(grads, R, n, ld, w, v, lr, mu, avg, max_blocks, s, fg);
    if (mom) {
        if (wavg) return avg_update_launch<true, true, true>(grads, R, n, ld, w, v, lr, mu, avg, max_blocks, s, fg);
        return avg_update_launch<true, false, true>(grads, R, n, ld, w, v, lr, mu, avg, max_blocks, s, fg);
    }
    if (wavg) return avg_update_launch<false, true, true>(grads, R, n, ld, w, v, lr, mu, avg, max_blocks, s, fg);
    return avg_update_launch<false, false, true>(grads, R, n, ld, w, v, lr, mu, avg, max_blocks, s, fg);
}

__global__ void set_int_kernel(int* p, int value)
{
    if (threadIdx.x == 0) *p = value;
}

hipError_t set_flag(int* p, int value, hipStream_t s)
{
    hipLaunchKernelGGL(set_int_kernel, dim3(1), dim3(64), 0, s, p, value);
    return hipGetLastError();
}


// ---- gradient average + Adam or AdaGrad ----------------------------------------------------
//
// The average g, summed in double in ascending r and divided by R before one rounding to float,
// followed by an adaptive update:
//   Adam (Kingma and Ba):  m = b1*m + (1-b1)*g;  v = b2*v + (1-b2)*g^2;
//                          w = w - lr * (m / (1 - b1^t)) / (sqrt(v / (1 - b2^t)) + eps)
//   AdaGrad (Duchi et al.): G = G + g^2;  w = w - lr * g / (sqrt(G) + eps)
// The update divides by a square root of squared averages, so where the average nearly cancels
// (|g| near eps) its absolute rounding error would be amplified into the step; the double sum of
// at most a few dozen floats is exact in practice, so g is the correctly rounded average.  The
// update itself is fp32 with correctly rounded division and square root; the bias corrections
// enter as their reciprocals, computed on the host in double.  Four consecutive elements per
// thread when every row and state vector is 16-byte aligned.

template <bool ADAM>
__device__ __forceinline__ void adapt_apply(float g, float& w, float& s1, float& s2,
                                            const AdaptParams& p)
{
    if (ADAM) {
        const float m = fmaf(p.b1, s1, p.c1 * g);
        const float v = fmaf(p.b2, s2, p.c2 * (g * g));
        s1 = m;
        s2 = v;
        w = fmaf(-p.lr, (m * p.ib1) / (sqrtf(v * p.ib2) + p.eps), w);
    } else {
        const float G = fmaf(g, g, s1);
        s1 = G;
        w = fmaf(-p.lr, g / (sqrtf(G) + p.eps), w);
    }
}

template <bool ADAM, bool AVG>
__device__ __forceinline__ void adapt_one(const float* __restrict__ grads, int R, long long ld,
                                          long long i, const AdaptParams& p)
{
    double s = (double)grads[i];
    for (int r = 1; r < R; ++r) s += (double)grads[(long long)r * ld + i];
    const float g = (float)(s / (double)R);
    if (AVG) p.avg[i] = g;
    float w = p.w[i], s1 = p.s1[i], s2 = ADAM ? p.s2[i] : 0.f;
    adapt_apply<ADAM>(g, w, s1, s2, p);
    p.w[i] = w;
    p.s1[i] = s1;
    if (ADAM) p.s2[i] = s2;
}

// n elements: threads below n / 4 take four each; the next one takes the n % 4 left over.
template <int RT, bool ADAM, bool AVG>
__global__ __launch_bounds__(256) void avg_adapt_vec4(const float* __restrict__ grads, int Rrt,
                                                      long long n, long long ld,
                                                      const AdaptParams p)
{
    const long long n4 = n / 4;
    const int R = RT > 0 ? RT : Rrt;
    for (long long t = (long long)blockIdx.x * 256 + threadIdx.x; t <= n4;
         t += (long long)gridDim.x * 256) {
        if (t == n4) {
            for (long long i = 4 * n4; i < n; ++i) adapt_one<ADAM, AVG>(grads, R, ld, i, p);
            break;
        }
        const f32x4* g4 = reinterpret_cast<const f32x4*>(grads) + t;
        const long long ld4 = ld / 4;
        const f32x4 g0 = __builtin_nontemporal_load(g4);
        double s[4] = {(double)g0[0], (double)g0[1], (double)g0[2], (double)g0[3]};
        if (RT > 0) {
            f32x4 buf[RT > 1 ? RT - 1 : 1];
#pragma unroll
            for (int r = 1; r < RT; ++r) buf[r - 1] = __builtin_nontemporal_load(g4 + r * ld4);
#pragma unroll
            for (int r = 1; r < RT; ++r)
#pragma unroll
                for (int j = 0; j < 4; ++j) s[j] += (double)buf[r - 1][j];
        } else {
            for (int r = 1; r < R; ++r) {
                const f32x4 x = __builtin_nontemporal_load(g4 + r * ld4);
#pragma unroll
                for (int j = 0; j < 4; ++j) s[j] += (double)x[j];
            }
        }
        const double dr = (double)R;
        const f32x4 g = {(float)(s[0] / dr), (float)(s[1] / dr), (float)(s[2] / dr),
                         (float)(s[3] / dr)};
        if (AVG) __builtin_nontemporal_store(g, reinterpret_cast<f32x4*>(p.avg) + t);
        f32x4 wv = reinterpret_cast<f32x4*>(p.w)[t];
        f32x4 a1 = reinterpret_cast<f32x4*>(p.s1)[t];
        f32x4 a2 = ADAM ? reinterpret_cast<f32x4*>(p.s2)[t] : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            float wj = wv[j], x1 = a1[j], x2 = a2[j];
            adapt_apply<ADAM>(g[j], wj, x1, x2, p);
            wv[j] = wj;
            a1[j] = x1;
            a2[j] = x2;
        }
        reinterpret_cast<f32x4*>(p.w)[t] = wv;
        reinterpret_cast<f32x4*>(p.s1)[t] = a1;
        if (ADAM) reinterpret_cast<f32x4*>(p.s2)[t] = a2;
    }
}

template <bool ADAM, bool AVG>
__global__ __launch_bounds__(256) void avg_adapt_scalar(const float* __restrict__ grads, int R,
                                                        long long n, long long ld,
                                                        const AdaptParams p)
{
    const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
    if (i >= n) return;
    adapt_one<ADAM, AVG>(grads, R, ld, i, p);
}

template <bool ADAM, bool AVG>
static hipError_t avg_adapt_launch(const float* grads, int R, size_t n, size_t ld,
                                   const AdaptParams& p, hipStream_t s, unsigned max_blocks)
{
    auto al = [](const void* q) { return (reinterpret_cast<uintptr_t>(q) & 15) == 0; };
    const bool vec = (ld % 4 == 0) && al(grads) && al(p.w) && al(p.s1) && (!ADAM || al(p.s2)) &&
                     (!AVG || al(p.avg));
    const long long nn = (long long)n, ll = (long long)ld;
    if (vec) {
        dim3 grid(grid_for(n / 4 + 1, 512));
        if (max_blocks && grid.x > max_blocks) grid.x = max_blocks;
        const size_t lds = max_blocks ? 0 : kStreamLds;
        switch (R) {
        case 1: hipLaunchKernelGGL((avg_adapt_vec4<1, ADAM, AVG>), grid, dim3(256), lds, s, grads, R, nn, ll, p); break;
        case 2: hipLaunchKernelGGL((avg_adapt_vec4<2, ADAM, AVG>), grid, dim3(256), lds, s, grads, R, nn, ll, p); break;
        case 4: hipLaunchKernelGGL((avg_adapt_vec4<4, ADAM, AVG>), grid, dim3(256), lds, s, grads, R, nn, ll, p); break;
        case 8: hipLaunchKernelGGL((avg_adapt_vec4<8, ADAM, AVG>), grid, dim3(256), lds, s, grads, R, nn, ll, p); break;
        case 16: hipLaunchKernelGGL((avg_adapt_vec4<16, ADAM, AVG>), grid, dim3(256), lds, s, grads, R, nn, ll, p); break;
        default: hipLaunchKernelGGL((avg_adapt_vec4<0, ADAM, AVG>), grid, dim3(256), lds, s, grads, R, nn, ll, p); break;
        }
    } else {
        hipLaunchKernelGGL((avg_adapt_scalar<ADAM, AVG>), dim3(grid_for(n, 256)), dim3(256), 0, s,
                           grads, R, nn, ll, p);
    }
    return hipGetLastError();
}

hipError_t average_adapt(const float* grads, int R, size_t n, size_t ld, bool adam,
                         const AdaptParams& p, hipStream_t s, unsigned max_blocks)
{
    if (adam) {
        if (p.avg) return avg_adapt_launch<true, true>(grads, R, n, ld, p, s, max_blocks);
        return avg_adapt_launch<true, false>(grads, R, n, ld, p, s, max_blocks);
    }
    if (p.avg) return avg_adapt_launch<false, true>(grads, R, n, ld, p, s, max_blocks);
    return avg_adapt_launch<false, false>(grads, R, n, ld, p, s, max_blocks);
}

}  // namespace mtx
