// Weight preparation, device side (see PrepJob): the work of one block of the preparation
// launch.  Shared by the preparation kernel and by a launch that carries the preparation blocks
// after its own (the direct first convolution's forward).
#pragma once

#include "device_common.h"
#include "internal.h"

namespace mtx {

constexpr int kPrepPerThread = 8, kPrepPerBlock = 256 * kPrepPerThread;

__device__ __forceinline__ unsigned prep_fdivu(const FastDiv& f, unsigned n)
{
    return (__umulhi(n, f.m) + n) >> f.s;
}

__device__ __forceinline__ int prep_src(const PrepJob& j, unsigned d)
{
    switch (j.kind) {
    case PREP_CONV_F: {  // d = co*(KK*cg) + uv*cg + ci
        const unsigned co = prep_fdivu(j.f0, d), r = d - co * (unsigned)(j.KK * j.cg);
        const unsigned uv = prep_fdivu(j.f1, r), ci = r - uv * (unsigned)j.cg;
        return ((int)co * j.cg + (int)ci) * j.KK + (int)uv;
    }
    case PREP_CONV_D: {  // d = ((g*cg + ci)*KK + uv)*og + co
        const unsigned r1 = prep_fdivu(j.f0, d), co = d - r1 * (unsigned)j.og;
        const unsigned r2 = prep_fdivu(j.f1, r1), uv = r1 - r2 * (unsigned)j.KK;
        const unsigned g = prep_fdivu(j.f2, r2), ci = r2 - g * (unsigned)j.cg;
        return (((int)g * j.og + (int)co) * j.cg + (int)ci) * j.KK + (int)uv;
    }
    case PREP_CONV_C: {  // d = ((g*KK + uv)*cg + ci)*og + co
        const unsigned r1 = prep_fdivu(j.f0, d), co = d - r1 * (unsigned)j.og;
        const unsigned r2 = prep_fdivu(j.f1, r1), ci = r1 - r2 * (unsigned)j.cg;
        const unsigned g = prep_fdivu(j.f2, r2), uv = r2 - g * (unsigned)j.KK;
        return (((int)g * j.og + (int)co) * j.cg + (int)ci) * j.KK + (int)uv;
    }
    case PREP_CONV_RUN: {  // d = (co*K + u)*RUN + j, j = v*Cp + ci; -1 for padding taps
        const unsigned r = prep_fdivu(j.f0, d), jj = d - r * (unsigned)j.RUN;
        const unsigned co = r / (unsigned)j.K, u = r - co * (unsigned)j.K;
        const unsigned v = prep_fdivu(j.f1, jj), ci = jj - v * (unsigned)j.Cp;
        if (v >= (unsigned)j.K || ci >= (unsigned)j.C) return -1;
        return (((int)co * j.C + (int)ci) * j.K + (int)u) * j.K + (int)v;
    }
    case PREP_FC_PERM: {  // d = o*IN + hw*C + c
        const unsigned o = prep_fdivu(j.f0, d), r = d - o * (unsigned)j.IN;
        const unsigned hw = prep_fdivu(j.f1, r), c = r - hw * (unsigned)j.C;
        return (int)o * j.IN + (int)c * j.HW + (int)hw;
    }
    default:
        return (int)d;
    }
}

// Block bid of the preparation launch (256 threads).
template <typename T>
__device__ __forceinline__ void prep_block(const PrepJob* __restrict__ jobs, int njobs,
                                           const float* __restrict__ w, T* __restrict__ dst,
                                           int bid)
{
    int jx = 0;
    for (int k = 1; k < njobs; ++k)
        if (jobs[k].block0 <= bid) jx = k;
    const PrepJob j = jobs[jx];
    const float* src = w + j.src;
    T* out = dst + j.dst;  // 16-byte aligned
    if (j.kind == PREP_CAST) {
        // plain conversion: 8 consecutive elements per thread, read 16 or 8 bytes at a time as
        // the source's alignment allows (a layer's weights start anywhere in the flat vector),
        // written with 16-byte stores
        static_assert(kPrepPerThread == 8, "cast step");
        const int d = (bid - j.block0) * kPrepPerBlock + (int)threadIdx.x * 8;
        if (d + 8 <= j.n) {
            float f[8];
            if (((uintptr_t)src & 15) == 0) {
                const float4 lo = *reinterpret_cast<const float4*>(src + d);
                const float4 hi = *reinterpret_cast<const float4*>(src + d + 4);
                f[0] = lo.x; f[1] = lo.y; f[2] = lo.z; f[3] = lo.w;
                f[4] = hi.x; f[5] = hi.y; f[6] = hi.z; f[7] = hi.w;
            } else if (((uintptr_t)src & 7) == 0) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float2 t = *reinterpret_cast<const float2*>(src + d + 2 * i);
                    f[2 * i] = t.x;
                    f[2 * i + 1] = t.y;
                }
            } else {
#pragma unroll
                for (int i = 0; i < 8; ++i) f[i] = src[d + i];
            }
            T v[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) v[i] = from_f32<T>(f[i]);
            uint4* o = reinterpret_cast<uint4*>(out + d);
            o[0] = reinterpret_cast<const uint4*>(v)[0];
            if constexpr (sizeof(T) == 4) o[1] = reinterpret_cast<const uint4*>(v)[1];
        } else {
            for (int i = d; i < j.n; ++i) out[i] = from_f32<T>(src[i]);
        }
        return;
    }
    const int base = (bid - j.block0) * kPrepPerBlock + threadIdx.x;
#pragma unroll
    for (int e = 0; e < kPrepPerThread; ++e) {
        const int d = base + e * 256;
        if (d < j.n) {
            const int si = prep_src(j, (unsigned)d);
            out[d] = from_f32<T>(si >= 0 ? src[si] : 0.f);
        }
    }
}

}  // namespace mtx
