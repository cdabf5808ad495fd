// Data-gradient launches: convolution (implicit GEMM, or col GEMM + col2im) and fully
// connected.
#include "igemm_ops.h"

namespace mtx {

// dx (NHWC) = sum over (u, v) in ascending order of col[g][(n, oh, ow)][(u, v, ci')] with
// oh*stride = h + pad - u (likewise for columns), times the ReLU mask of the layer below.
// One thread per element of dx, channels fastest.  KT > 0: kernel size known at compile time
// and stride 1.
template <typename T, int KT>
__global__ __launch_bounds__(256) void col2im_kernel(const GemmArgs a, const float* __restrict__ col)
{
    const int t = blockIdx.x * 256 + threadIdx.x;
    const int total = a.N * a.C * a.H * a.W;
    if (t >= total) return;
    const unsigned pos = fdiv(a.fd_c, (unsigned)t), ci = (unsigned)t - pos * (unsigned)a.C;
    const unsigned b = fdiv(a.fd_hw, pos), hw = pos - b * (unsigned)(a.H * a.W);
    const unsigned hq = fdiv(a.fd_w, hw);
    const int h = (int)hq, w = (int)(hw - hq * (unsigned)a.W);
    const int grp = (int)ci / a.cg, cl = (int)ci - grp * a.cg;
    const long long Q = (long long)a.N * a.OH * a.OW, P = (long long)a.KK * a.cg;
    const float* cp = col + (long long)grp * Q * P + (long long)b * a.OH * a.OW * P + cl;
    float acc = 0.f;
    if constexpr (KT > 0) {
#pragma unroll
        for (int u = 0; u < KT; ++u) {
            const int oh = h + a.PD - u;
            const bool okh = (unsigned)oh < (unsigned)a.OH;
#pragma unroll
            for (int v = 0; v < KT; ++v) {
                const int ow = w + a.PD - v;
                const bool ok = okh && (unsigned)ow < (unsigned)a.OW;
                const float x = cp[ok ? ((long long)oh * a.OW + ow) * P + (u * KT + v) * a.cg : 0];
                acc += ok ? x : 0.f;
            }
        }
    } else {
        for (int u = 0; u < a.K; ++u) {
            const int th = h + a.PD - u;
            if (th < 0) break;
            const int oh = th / a.S;
            if (oh * a.S != th || oh >= a.OH) continue;
            for (int v = 0; v < a.K; ++v) {
                const int tw = w + a.PD - v;
                if (tw < 0) break;
                const int ow = tw / a.S;
                if (ow * a.S != tw || ow >= a.OW) continue;
                acc += cp[((long long)oh * a.OW + ow) * P + (u * a.K + v) * a.cg];
            }
        }
    }
    if (a.mask) {
        const float m = a.mask_f32 ? static_cast<const float*>(a.mask)[t]
                                   : to_f32<T>(static_cast<const T*>(a.mask)[t]);
        if (!(m > 0.f)) acc = 0.f;
    }
    static_cast<T*>(a.out)[t] = from_f32<T>(acc);
}

// Four channels per thread (C and C/G multiples of 4, so that the four share a group and every
// col row, dx row and mask row access is 16-byte aligned); the same taps in the same order as
// col2im_kernel.  KT, ST > 0: kernel size and stride known at compile time (0: from a).
template <typename T>
__device__ __forceinline__ void load4(const void* p, long long i, float (&v)[4])
{
    if constexpr (sizeof(T) == 4) {
        const float4 q = *reinterpret_cast<const float4*>(static_cast<const float*>(p) + i);
        v[0] = q.x; v[1] = q.y; v[2] = q.z; v[3] = q.w;
    } else {
        const uint2 q = *reinterpret_cast<const uint2*>(static_cast<const bf16_t*>(p) + i);
        v[0] = bf16_to_f32((bf16_t)(q.x & 0xffffu)); v[1] = bf16_to_f32((bf16_t)(q.x >> 16));
        v[2] = bf16_to_f32((bf16_t)(q.y & 0xffffu)); v[3] = bf16_to_f32((bf16_t)(q.y >> 16));
    }
}

template <typename T, int KT, int ST>
__global__ __launch_bounds__(256) void col2im_vec4_kernel(const GemmArgs a, const float* __restrict__ col)
{
    const long long t = (long long)blockIdx.x * 256 + threadIdx.x;
    const long long total = (long long)a.N * a.C * a.H * a.W / 4;
    if (t >= total) return;
    const unsigned e = (unsigned)t * 4u;
    const unsigned pos = fdiv(a.fd_c, e), ci = e - pos * (unsigned)a.C;
    const unsigned b = fdiv(a.fd_hw, pos), hw = pos - b * (unsigned)(a.H * a.W);
    const unsigned hq = fdiv(a.fd_w, hw);
    const int h = (int)hq, w = (int)(hw - hq * (unsigned)a.W);
    const int grp = (int)ci / a.cg, cl = (int)ci - grp * a.cg;
    const int K = KT > 0 ? KT : a.K, S = ST > 0 ? ST : a.S;
    const long long Q = (long long)a.N * a.OH * a.OW, P = (long long)K * K * a.cg;
    const float* cp = col + (long long)grp * Q * P + (long long)b * a.OH * a.OW * P + cl;
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    for (int u = 0; u < K; ++u) {
        const int th = h + a.PD - u;
        const int oh = th / S;
        if (th < 0 || oh * S != th || oh >= a.OH) continue;
        for (int v = 0; v < K; ++v) {
            const int tw = w + a.PD - v;
            const int ow = tw / S;
            if (tw < 0 || ow * S != tw || ow >= a.OW) continue;
            const f32x4 x = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(
                cp + ((long long)oh * a.OW + ow) * P + (u * K + v) * a.cg));
            acc[0] += x[0]; acc[1] += x[1]; acc[2] += x[2]; acc[3] += x[3];
        }
    }
    if (a.mask) {
        float m[4];
        if (a.mask_f32) load4<float>(a.mask, (long long)e, m);
        else load4<T>(a.mask, (long long)e, m);
#pragma unroll
        for (int i = 0; i < 4; ++i)
            if (!(m[i] > 0.f)) acc[i] = 0.f;
    }
    if constexpr (sizeof(T) == 4) {
        *reinterpret_cast<float4*>(static_cast<float*>(a.out) + e) =
            make_float4(acc[0], acc[1], acc[2], acc[3]);
    } else {
        uint2 q;
        q.x = (unsigned)f32_to_bf16(acc[0]) | ((unsigned)f32_to_bf16(acc[1]) << 16);
        q.y = (unsigned)f32_to_bf16(acc[2]) | ((unsigned)f32_to_bf16(acc[3]) << 16);
        *reinterpret_cast<uint2*>(static_cast<bf16_t*>(a.out) + e) = q;
    }
}

template <typename T>
static void launch_col2im(const GemmArgs& c, const float* col, hipStream_t s)
{
    const long long total = (long long)c.N * c.C * c.H * c.W;
    if (c.C % 4 == 0 && c.cg % 4 == 0 && total < (1ll << 32)) {
        dim3 grid((unsigned)((total / 4 + 255) / 256));
        if (c.S == 1 && c.K == 3) hipLaunchKernelGGL((col2im_vec4_kernel<T, 3, 1>), grid, dim3(256), 0, s, c, col);
        else if (c.S == 1 && c.K == 5) hipLaunchKernelGGL((col2im_vec4_kernel<T, 5, 1>), grid, dim3(256), 0, s, c, col);
        else if (c.S == 2 && c.K == 3) hipLaunchKernelGGL((col2im_vec4_kernel<T, 3, 2>), grid, dim3(256), 0, s, c, col);
        else if (c.S == 2 && c.K == 1) hipLaunchKernelGGL((col2im_vec4_kernel<T, 1, 2>), grid, dim3(256), 0, s, c, col);
        else hipLaunchKernelGGL((col2im_vec4_kernel<T, 0, 0>), grid, dim3(256), 0, s, c, col);
        return;
    }
    dim3 grid((unsigned)((total + 255) / 256));
    if (c.S == 1 && c.K == 3) hipLaunchKernelGGL((col2im_kernel<T, 3>), grid, dim3(256), 0, s, c, col);
    else if (c.S == 1 && c.K == 5) hipLaunchKernelGGL((col2im_kernel<T, 5>), grid, dim3(256), 0, s, c, col);
    else hipLaunchKernelGGL((col2im_kernel<T, 0>), grid, dim3(256), 0, s, c, col);
}

hipError_t conv_dgrad(Dt dt, const ConvGeom& g, const void* dy, const void* wd, void* dx,
                      const void* mask, bool mask_f32, float* partial, hipStream_t s)
{
    GemmArgs a = conv_args(g);
    a.a = dy; a.b = wd; a.out = dx; a.mask = mask; a.mask_f32 = mask_f32;
    a.vec_out = g.C % 4 == 0 && a.cg % 4 == 0;
    const unsigned es = dt == DT_F32 ? 4 : 2;
    a.a_bytes = (unsigned)((size_t)g.N * g.OC * g.OH * g.OW * es);
    a.b_bytes = (unsigned)((size_t)g.OC * a.cg * a.KK * es);
    const GemmDims d = conv_dgrad_dims(dt, g);
    a.Pdim = d.P; a.Qdim = d.Q; a.Kdim = d.K;
    const GemmPlan p = plan_for(dt, d);
    const bool v = a.og % vec_elems(dt) == 0;  // then OC and Kdim are multiples too
    if (g.S == 1) {
        if (dt == DT_F32) {
            if (v) return run_gemm<ConvDgrad<float, true>, L_KD, L_KD>(a, p, d.Z, partial, s);
            return run_gemm<ConvDgrad<float, true>, L_SK, L_SR>(a, p, d.Z, partial, s);
        }
        if (v) return run_gemm<ConvDgrad<bf16_t, true>, L_KV, L_KV>(a, p, d.Z, partial, s);
        return run_gemm<ConvDgrad<bf16_t, true>, L_SK, L_SR>(a, p, d.Z, partial, s);
    }
    if (dt == DT_F32) return run_gemm<ConvDgrad<float, false>, L_SK, L_SR>(a, p, d.Z, partial, s);
    return run_gemm<ConvDgrad<bf16_t, false>, L_SK, L_SR>(a, p, d.Z, partial, s);
}

hipError_t conv_dgrad_col(Dt dt, const ConvGeom& g, const void* dy, const void* wc, void* dx,
                          const void* mask, bool mask_f32, float* col,
                          float* partial, hipStream_t s)
{
    GemmArgs a = conv_args(g);
    a.a = dy; a.b = wc; a.out = col;
    a.vec_out = (a.KK * a.cg) % 4 == 0;
    const unsigned es = dt == DT_F32 ? 4 : 2;
    a.a_bytes = (unsigned)((size_t)g.N * g.OC * g.OH * g.OW * es);
    a.b_bytes = (unsigned)((size_t)g.OC * a.cg * a.KK * es);
    const GemmDims d = conv_dgrad_col_dims(dt, g);
    a.Pdim = d.P; a.Qdim = d.Q; a.Kdim = d.K;
    const GemmPlan p = plan_for(dt, d);
    const bool v = a.og % vec_elems(dt) == 0;
    hipError_t e;
    if (dt == DT_F32)
        e = v ? run_gemm<ConvDgradCol<float>, L_KD, L_KD>(a, p, d.Z, partial, s)
              : run_gemm<ConvDgradCol<float>, L_SK, L_SK>(a, p, d.Z, partial, s);
    else
        e = v ? run_gemm<ConvDgradCol<bf16_t>, L_KV, L_KV>(a, p, d.Z, partial, s)
              : run_gemm<ConvDgradCol<bf16_t>, L_SK, L_SK>(a, p, d.Z, partial, s);
    if (e != hipSuccess) return e;
    timing_split(s, "col2im");
    GemmArgs c = conv_args(g);
    c.out = dx; c.mask = mask; c.mask_f32 = mask_f32;
    if (dt == DT_F32) launch_col2im<float>(c, col, s);
    else launch_col2im<bf16_t>(c, col, s);
    return hipGetLastError();
}

hipError_t fc_dgrad(Dt dt, int B, int IN, int OUT, const void* dy, const void* w, void* dx,
                    const void* mask, bool mask_f32, float* partial, hipStream_t s)
{
    GemmArgs a{};
    a.a = dy; a.b = w; a.out = dx; a.mask = mask; a.mask_f32 = mask_f32;
    a.N = B; a.C = IN; a.OC = OUT; a.G = 1; a.R = 1; a.perm_c = 1; a.perm_hw = 1;
    a.vec_out = IN % 4 == 0;
    const unsigned es = dt == DT_F32 ? 4 : 2;
    a.a_bytes = (unsigned)((size_t)B * OUT * es);
    a.b_bytes = (unsigned)((size_t)OUT * IN * es);
    const GemmDims d = fc_dgrad_dims(dt, B, IN, OUT);
    a.Pdim = d.P; a.Qdim = d.Q; a.Kdim = d.K;
    const GemmPlan p = plan_for(dt, d);
    const bool pv = IN % vec_elems(dt) == 0, qv = OUT % vec_elems(dt) == 0;
    if (dt == DT_F32) {
        typedef FcDgrad<float> Op;
        if (pv && qv) return run_gemm<Op, L_RT, L_KD>(a, p, d.Z, partial, s);
        if (pv) return run_gemm<Op, L_RT, L_SK>(a, p, d.Z, partial, s);
        if (qv) return run_gemm<Op, L_SR, L_KD>(a, p, d.Z, partial, s);
        return run_gemm<Op, L_SR, L_SK>(a, p, d.Z, partial, s);
    }
    typedef FcDgrad<bf16_t> Op;
    if (pv && qv) return run_gemm<Op, L_RT, L_KV>(a, p, d.Z, partial, s);
    if (pv) return run_gemm<Op, L_RT, L_SK>(a, p, d.Z, partial, s);
    if (qv) return run_gemm<Op, L_SR, L_KV>(a, p, d.Z, partial, s);
    return run_gemm<Op, L_SR, L_SK>(a, p, d.Z, partial, s);
}

}  // namespace mtx
