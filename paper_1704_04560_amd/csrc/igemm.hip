// Implicit-GEMM kernels on the gfx950 matrix cores for the convolution and fully connected
// layers: forward (+bias, +ReLU), data gradient (+ReLU mask of the layer below) and weight
// gradient per shard (with the bias gradient as one extra output column).
//
// Every operation is C[p][q] = sum_k P[p][k] * Q[q][k].  One kernel template stages BP x BK
// and BQ x BK tiles in LDS (k contiguous within a row, rows padded by 16 bytes) and runs 16x16
// MFMA fragments over them:
//   fp32: v_mfma_f32_16x16x4_f32, four per 16-byte LDS read (lane group g feeds k = 4g + t to
//         the t-th instruction for both operands, so the product is unchanged);
//   bf16: v_mfma_f32_16x16x32_bf16, one per 16-byte read (8 values per lane).
// 256 threads = 4 waves in a 2 x 2 grid; a wave owns FP x FQ fragments of 16 x 16.  The MFMA
// output layout (lane l, register v -> row 4*(l/16) + v, column l%16) makes consecutive lanes
// walk consecutive q, the contiguous dimension of every output.
//
// Operand loading.  An operand tile is BR rows x BK reduction steps.  It is loaded either
// "row-fast" (consecutive threads take consecutive rows, each thread keeps one row for the whole
// kernel and steps through k) or "k-fast" (consecutive threads take consecutive k, each thread
// keeps one k per tile and steps through rows); the choice follows the contiguous dimension in
// memory.  Whatever is fixed per thread is decoded once; the part of the convolution index map
// that varies per element comes from a table in LDS built at kernel start, so the inner loop
// does no integer division.
//
// Reduction splits.  When a problem has too few output tiles to fill the GPU, the reduction is
// split over blockIdx.z; every split writes fp32 partial sums and a second kernel adds them in
// ascending split order and applies the operation's epilogue (deterministic, no atomics).
#include "device_common.h"
#include "internal.h"

namespace mtx {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

template <typename T> struct Mma;

template <> struct Mma<float> {
    typedef f32x4 frag;
    static constexpr int VEC = 4;     // elements per 16-byte lane read
    static constexpr int KSTEP = 16;  // k covered by one read across the 4 lane groups
    __device__ __forceinline__ static void run(f32x4& acc, const frag& a, const frag& b)
    {
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[0], b[0], acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[1], b[1], acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[2], b[2], acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[3], b[3], acc, 0, 0, 0);
    }
};

template <> struct Mma<bf16_t> {
    typedef s16x8 frag;
    static constexpr int VEC = 8;
    static constexpr int KSTEP = 32;
    __device__ __forceinline__ static void run(f32x4& acc, const frag& a, const frag& b)
    {
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                      __builtin_bit_cast(bf16x8, b), acc, 0,
                                                      0, 0);
    }
};

template <typename T> __device__ __forceinline__ T zero() { return T(0); }
template <typename T> __device__ __forceinline__ T one();
template <> __device__ __forceinline__ float one<float>() { return 1.0f; }
template <> __device__ __forceinline__ bf16_t one<bf16_t>() { return (bf16_t)0x3f80; }

// One entry of an index table: a flat offset and the two kernel-window coordinates it stands
// for (needed for the zero-padding test).
struct TabEnt {
    int off;
    short u, v;
};

constexpr int kMaxTab = 4096;  // largest reduction length with an LDS table (32 KB)

struct Ctx {
    int grp, r, split, kbeg, kend, b0;
    const TabEnt* tab;  // LDS table (operation specific), or null
};

__device__ __forceinline__ void decode_z(const GemmArgs& a, Ctx& c)
{
    const int z = blockIdx.z;
    c.grp = z % a.G;
    const int rest = z / a.G;
    c.r = rest / a.splits;
    c.split = rest - c.r * a.splits;
    c.kbeg = c.split * a.kchunk;
    c.kend = min(a.Kdim, c.kbeg + a.kchunk);
    c.b0 = c.r * a.N;
    c.tab = nullptr;
}

// Operand reads go through raw buffer loads: the buffer resource carries the tensor's size in
// bytes and the hardware returns 0 for any offset at or past it.  Zero padding and tile tails
// therefore only select an out-of-range offset (kOOB); there is no branch, and no index can read
// outside its tensor.
constexpr unsigned kOOB = 0x80000000u;     // every tensor is smaller than 2 GiB
constexpr unsigned kRsrcWord3 = 0x00020000u;  // raw buffer, 32-bit data format

template <typename T> struct Buf {
    __amdgpu_buffer_rsrc_t r;
    __device__ __forceinline__ Buf(const void* p, unsigned bytes)
        : r(__builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes,
                                              (int)kRsrcWord3))
    {
    }
    __device__ __forceinline__ T at(bool ok, int idx) const
    {
        const int off = ok ? idx * (int)sizeof(T) : (int)kOOB;
        if constexpr (sizeof(T) == 4)
            return __builtin_bit_cast(T, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
        else
            return __builtin_bit_cast(T, __builtin_amdgcn_raw_buffer_load_b16(r, off, 0, 0));
    }
};

constexpr int kFar = 1 << 14;  // window coordinate that fails every bounds test

// ------------------------------------------------------------------------------------------
// Convolution forward: p = output channel in the group, q = (image, oh, ow),
// k = (input channel in the group, u, v).  P = weights (k-fast), Q = input patches (row-fast,
// table over k).
// ------------------------------------------------------------------------------------------
template <typename T> struct ConvFwd {
    typedef T TT;
    static constexpr bool P_IS_A = false;
    static constexpr bool P_ROW_FAST = false, Q_ROW_FAST = true;
    static constexpr bool KTAB = true, QTAB = false;
    __device__ static TabEnt ktab_entry(const GemmArgs& a, const Ctx& c, int k)
    {
        if (k >= c.kend) return TabEnt{0, (short)kFar, (short)kFar};
        const unsigned ci = (unsigned)k / a.KK, rr = (unsigned)k - ci * a.KK;
        const unsigned u = rr / a.K, v = rr - u * a.K;
        return TabEnt{(int)((ci * a.H + u) * a.W + v), (short)u, (short)v};
    }
    struct PK { int base; bool ok; };
    __device__ static PK pk(const GemmArgs& a, const Ctx& c, int k)
    {
        return PK{c.grp * a.og * a.Kdim + k, k < c.kend};
    }
    __device__ static T p_at(const GemmArgs& a, const Buf<T>& B, const PK& s, int p)
    {
        return B.at(s.ok && p < a.Pdim, s.base + p * a.Kdim);
    }
    struct QR { int base, h0, w0; };
    __device__ static QR qr(const GemmArgs& a, const Ctx& c, int q)
    {
        QR s;
        const unsigned ohw = a.OH * a.OW;
        const bool ok = q < a.Qdim;
        const unsigned qq = ok ? q : 0;
        const unsigned b = qq / ohw, hw = qq - b * ohw, ho = hw / a.OW, wo = hw - ho * a.OW;
        s.h0 = ok ? (int)(ho * a.S) - a.PD : -kFar;
        s.w0 = (int)(wo * a.S) - a.PD;
        s.base = (int)(b * a.C + c.grp * a.cg) * a.H * a.W + s.h0 * a.W + s.w0;
        return s;
    }
    template <bool TAB>
    __device__ static T q_at(const GemmArgs& a, const Buf<T>& B, const Ctx& c, const QR& s, int k)
    {
        const TabEnt e = TAB ? c.tab[k - c.kbeg] : ktab_entry(a, c, k);
        const int hi = s.h0 + e.u, wi = s.w0 + e.v;
        return B.at((unsigned)hi < (unsigned)a.H && (unsigned)wi < (unsigned)a.W, s.base + e.off);
    }
    __device__ static void store(const GemmArgs& a, const Ctx& c, int p, int q, float acc)
    {
        const int co = c.grp * a.og + p;
        const unsigned ohw = a.OH * a.OW;
        const unsigned b = (unsigned)q / ohw, hw = (unsigned)q - b * ohw;
        float v = acc + a.bias[co];
        if (a.relu) v = v > 0.f ? v : 0.f;
        const int idx = (int)(b * a.OC + co) * (int)ohw + (int)hw;
        if (a.out_f32) static_cast<float*>(a.out)[idx] = v;
        else static_cast<T*>(a.out)[idx] = from_f32<T>(v);
    }
};

// ------------------------------------------------------------------------------------------
// Convolution data gradient: p = input channel in the group, q = (image, h, w),
// k = (output channel in the group, u, v); dy[oh][ow] contributes where h = oh*stride - pad + u
// (likewise for columns).  P = weights (k-fast), Q = dy (row-fast).  STRIDE1: the table holds
// the offset of (co, -u, -v) and the test is 0 <= h + pad - u < OH; otherwise the divisibility by
// the stride is tested element by element.
// ------------------------------------------------------------------------------------------
template <typename T, bool STRIDE1> struct ConvDgrad {
    typedef T TT;
    static constexpr bool P_IS_A = false;
    static constexpr bool P_ROW_FAST = false, Q_ROW_FAST = true;
    static constexpr bool KTAB = STRIDE1, QTAB = false;
    __device__ static TabEnt ktab_entry(const GemmArgs& a, const Ctx& c, int k)
    {
        if (k >= c.kend) return TabEnt{0, (short)-kFar, (short)-kFar};
        const unsigned co = (unsigned)k / a.KK, rr = (unsigned)k - co * a.KK;
        const unsigned u = rr / a.K, v = rr - u * a.K;
        return TabEnt{(int)(co * a.OH * a.OW) - (int)(u * a.OW) - (int)v, (short)u, (short)v};
    }
    struct PK { int base; bool ok; };
    __device__ static PK pk(const GemmArgs& a, const Ctx& c, int k)
    {
        const unsigned co = (unsigned)k / a.KK, rr = (unsigned)k - co * a.KK;
        return PK{(int)((c.grp * a.og + co) * a.cg * a.KK + rr), k < c.kend};
    }
    __device__ static T p_at(const GemmArgs& a, const Buf<T>& B, const PK& s, int p)
    {
        return B.at(s.ok && p < a.Pdim, s.base + p * a.KK);
    }
    struct QR { int base, hp, wp; };
    __device__ static QR qr(const GemmArgs& a, const Ctx& c, int q)
    {
        QR s;
        const unsigned hw_in = a.H * a.W;
        const bool ok = q < a.Qdim;
        const unsigned qq = ok ? q : 0;
        const unsigned b = qq / hw_in, hw = qq - b * hw_in, h = hw / a.W, w = hw - h * a.W;
        s.hp = ok ? (int)h + a.PD : -kFar;
        s.wp = (int)w + a.PD;
        s.base = (int)(b * a.OC + c.grp * a.og) * a.OH * a.OW;
        if (STRIDE1) s.base += s.hp * a.OW + s.wp;
        return s;
    }
    template <bool TAB>
    __device__ static T q_at(const GemmArgs& a, const Buf<T>& B, const Ctx& c, const QR& s, int k)
    {
        if constexpr (STRIDE1) {
            const TabEnt e = TAB ? c.tab[k - c.kbeg] : ktab_entry(a, c, k);
            const int th = s.hp - e.u, tw = s.wp - e.v;
            return B.at((unsigned)th < (unsigned)a.OH && (unsigned)tw < (unsigned)a.OW,
                        s.base + e.off);
        } else {
            const unsigned co = (unsigned)k / a.KK, rr = (unsigned)k - co * a.KK;
            const int u = (int)(rr / a.K), v = (int)(rr - (rr / a.K) * a.K);
            const int th = s.hp - u, tw = s.wp - v;
            const int oh = th / a.S, ow = tw / a.S;
            const bool ok = k < c.kend && th >= 0 && tw >= 0 && oh * a.S == th &&
                            ow * a.S == tw && oh < a.OH && ow < a.OW;
            return B.at(ok, s.base + ((int)co * a.OH + oh) * a.OW + ow);
        }
    }
    __device__ static void store(const GemmArgs& a, const Ctx& c, int p, int q, float acc)
    {
        const int ci = c.grp * a.cg + p;
        const unsigned hw_in = a.H * a.W;
        const unsigned b = (unsigned)q / hw_in, hw = (unsigned)q - b * hw_in;
        const int idx = (int)(b * a.C + ci) * (int)hw_in + (int)hw;
        if (a.mask) {
            const float m = a.mask_f32 ? static_cast<const float*>(a.mask)[idx]
                                       : to_f32<T>(static_cast<const T*>(a.mask)[idx]);
            if (!(m > 0.f)) acc = 0.f;
        }
        static_cast<T*>(a.out)[idx] = from_f32<T>(acc);
    }
};

// ------------------------------------------------------------------------------------------
// Convolution weight gradient of one shard: p = output channel in the group,
// q = (input channel in the group, u, v) plus one extra column q = cg*K*K of ones that yields
// the bias gradient, k = (image in the shard, oh, ow).  Both operands k-fast; the q part of the
// patch offset comes from a per-block table.  blockIdx.z = (shard * splits + split) * G + group.
// ------------------------------------------------------------------------------------------
template <typename T> struct ConvWgrad {
    typedef T TT;
    static constexpr bool P_IS_A = true;
    static constexpr bool P_ROW_FAST = false, Q_ROW_FAST = false;
    static constexpr bool KTAB = false, QTAB = true;
    __device__ static TabEnt qtab_entry(const GemmArgs& a, int q)
    {
        if (q >= a.cg * a.KK) return TabEnt{0, (short)kFar, (short)kFar};
        const unsigned ci = (unsigned)q / a.KK, rr = (unsigned)q - ci * a.KK;
        const unsigned u = rr / a.K, v = rr - u * a.K;
        return TabEnt{(int)((ci * a.H + u) * a.W + v), (short)u, (short)v};
    }
    struct PK { int base; bool ok; };
    __device__ static PK pk(const GemmArgs& a, const Ctx& c, int k)
    {
        const unsigned ohw = a.OH * a.OW;
        const bool ok = k < c.kend;
        const unsigned kk = ok ? k : c.kbeg;
        const unsigned b = kk / ohw, hw = kk - b * ohw;
        return PK{(int)(((c.b0 + b) * a.OC + c.grp * a.og) * ohw + hw), ok};
    }
    __device__ static T p_at(const GemmArgs& a, const Buf<T>& B, const PK& s, int p)
    {
        return B.at(s.ok && p < a.Pdim, s.base + p * a.OH * a.OW);
    }
    struct QK { int base, h0, w0; bool ok; };
    __device__ static QK qk(const GemmArgs& a, const Ctx& c, int k)
    {
        QK s;
        const unsigned ohw = a.OH * a.OW;
        s.ok = k < c.kend;
        const unsigned kk = s.ok ? k : c.kbeg;
        const unsigned b = kk / ohw, hw = kk - b * ohw, ho = hw / a.OW, wo = hw - ho * a.OW;
        s.h0 = s.ok ? (int)(ho * a.S) - a.PD : -kFar;
        s.w0 = (int)(wo * a.S) - a.PD;
        s.base = (int)((c.b0 + b) * a.C + c.grp * a.cg) * a.H * a.W + s.h0 * a.W + s.w0;
        return s;
    }
    template <bool TAB>
    __device__ static T q_atk(const GemmArgs& a, const Buf<T>& B, const Ctx& c, const QK& s, int q,
                              int q0)
    {
        const TabEnt e = TAB ? c.tab[q - q0] : qtab_entry(a, q);
        const int hi = s.h0 + e.u, wi = s.w0 + e.v;
        const T v = B.at((unsigned)hi < (unsigned)a.H && (unsigned)wi < (unsigned)a.W,
                         s.base + e.off);
        return (q == a.cg * a.KK) ? (s.ok ? one<T>() : zero<T>()) : v;
    }
    __device__ static void store(const GemmArgs& a, const Ctx& c, int p, int q, float acc)
    {
        const int co = c.grp * a.og + p;
        const int nq = a.cg * a.KK;
        float* g = static_cast<float*>(a.out) + c.r * a.out_ld;
        if (q < nq) g[a.out_off + co * nq + q] = acc;
        else g[a.bias_off + co] = acc;
    }
};

// ------------------------------------------------------------------------------------------
// Convolution data gradient in two passes, for convolutions whose implicit data-gradient GEMM
// would spend much of its reduction on taps outside dy (unpadded convolutions): first
//   col[g][(ci, u, v)][(image, oh, ow)] = sum_co W[g*og + co][ci][u][v] * dy[image][g*og + co][oh][ow]
// as an exact GEMM (p = (ci, u, v), q = (image, oh, ow), k = co; both operands row-fast), then
// col2im_kernel gathers dx from it.  col is fp32, [G][cg*K*K][N*OH*OW].
// ------------------------------------------------------------------------------------------
template <typename T> struct ConvDgradCol {
    typedef T TT;
    static constexpr bool P_IS_A = false;
    static constexpr bool P_ROW_FAST = true, Q_ROW_FAST = true;
    static constexpr bool KTAB = false, QTAB = false;
    struct PR { int base; bool ok; };
    __device__ static PR pr(const GemmArgs& a, const Ctx& c, int p)
    {
        return PR{c.grp * a.og * a.cg * a.KK + p, p < a.Pdim};
    }
    __device__ static T p_atr(const GemmArgs& a, const Buf<T>& B, const Ctx& c, const PR& s, int k)
    {
        return B.at(s.ok && k < c.kend, s.base + k * a.cg * a.KK);
    }
    struct QR { int base; bool ok; };
    __device__ static QR qr(const GemmArgs& a, const Ctx& c, int q)
    {
        const unsigned ohw = a.OH * a.OW;
        const bool ok = q < a.Qdim;
        const unsigned qq = ok ? q : 0;
        const unsigned b = qq / ohw, hw = qq - b * ohw;
        return QR{(int)((b * a.OC + c.grp * a.og) * ohw + hw), ok};
    }
    template <bool TAB>
    __device__ static T q_at(const GemmArgs& a, const Buf<T>& B, const Ctx& c, const QR& s, int k)
    {
        return B.at(s.ok && k < c.kend, s.base + k * a.OH * a.OW);
    }
    __device__ static void store(const GemmArgs& a, const Ctx& c, int p, int q, float acc)
    {
        static_cast<float*>(a.out)[((long long)c.grp * a.Pdim + p) * a.Qdim + q] = acc;
    }
};

// dx[b][ci][h][w] = sum over (u, v) in ascending order of col[g][(ci', u, v)][(b, oh, ow)] with
// oh*stride = h + pad - u (likewise for columns), times the ReLU mask of the layer below.
// KT > 0: kernel size known at compile time, stride 1 (the loops unroll; no division).
template <typename T, int KT>
__global__ __launch_bounds__(256) void col2im_kernel(const GemmArgs a, const float* __restrict__ col)
{
    const int t = blockIdx.x * 256 + threadIdx.x;
    const int total = a.N * a.C * a.H * a.W;
    if (t >= total) return;
    const unsigned hw_in = a.H * a.W;
    const unsigned bc = (unsigned)t / hw_in, hw = (unsigned)t - bc * hw_in;
    const unsigned b = bc / a.C, ci = bc - b * a.C;
    const int h = (int)(hw / a.W), w = (int)(hw - (hw / a.W) * a.W);
    const unsigned grp = ci / a.cg, cl = ci - grp * a.cg;
    const long long Q = (long long)a.N * a.OH * a.OW;
    const float* cp = col + ((long long)grp * a.cg * a.KK + (long long)cl * a.KK) * Q +
                      (long long)b * a.OH * a.OW;
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
                const float x = cp[ok ? (long long)(u * KT + v) * Q + oh * a.OW + ow : 0];
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
                acc += cp[(long long)(u * a.K + v) * Q + oh * a.OW + ow];
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

template <typename T>
static void launch_col2im(const GemmArgs& c, const float* col, hipStream_t s)
{
    const long long total = (long long)c.N * c.C * c.H * c.W;
    dim3 grid((unsigned)((total + 255) / 256));
    if (c.S == 1 && c.K == 3) hipLaunchKernelGGL((col2im_kernel<T, 3>), grid, dim3(256), 0, s, c, col);
    else if (c.S == 1 && c.K == 5) hipLaunchKernelGGL((col2im_kernel<T, 5>), grid, dim3(256), 0, s, c, col);
    else hipLaunchKernelGGL((col2im_kernel<T, 0>), grid, dim3(256), 0, s, c, col);
}

// ------------------------------------------------------------------------------------------
// Fully connected layers
// ------------------------------------------------------------------------------------------

// Forward: p = sample, q = output unit, k = input feature.  Both operands k-fast.
template <typename T> struct FcFwd {
    typedef T TT;
    static constexpr bool P_IS_A = true;
    static constexpr bool P_ROW_FAST = false, Q_ROW_FAST = false;
    static constexpr bool KTAB = false, QTAB = false;
    struct PK { int k; bool ok; };
    __device__ static PK pk(const GemmArgs&, const Ctx& c, int k) { return PK{k, k < c.kend}; }
    __device__ static T p_at(const GemmArgs& a, const Buf<T>& B, const PK& s, int p)
    {
        return B.at(s.ok && p < a.Pdim, p * a.Kdim + s.k);
    }
    typedef PK QK;
    __device__ static QK qk(const GemmArgs&, const Ctx& c, int k) { return QK{k, k < c.kend}; }
    template <bool TAB>
    __device__ static T q_atk(const GemmArgs& a, const Buf<T>& B, const Ctx&, const QK& s, int q,
                              int)
    {
        return B.at(s.ok && q < a.Qdim, q * a.Kdim + s.k);
    }
    __device__ static void store(const GemmArgs& a, const Ctx&, int p, int q, float acc)
    {
        float v = acc + a.bias[q];
        if (a.relu) v = v > 0.f ? v : 0.f;
        const int idx = p * a.Qdim + q;
        if (a.out_f32) static_cast<float*>(a.out)[idx] = v;
        else static_cast<T*>(a.out)[idx] = from_f32<T>(v);
    }
};

// Data gradient: p = sample, q = input feature, k = output unit.  P k-fast, Q row-fast.
template <typename T> struct FcDgrad {
    typedef T TT;
    static constexpr bool P_IS_A = true;
    static constexpr bool P_ROW_FAST = false, Q_ROW_FAST = true;
    static constexpr bool KTAB = false, QTAB = false;
    struct PK { int k; bool ok; };
    __device__ static PK pk(const GemmArgs&, const Ctx& c, int k) { return PK{k, k < c.kend}; }
    __device__ static T p_at(const GemmArgs& a, const Buf<T>& B, const PK& s, int p)
    {
        return B.at(s.ok && p < a.Pdim, p * a.Kdim + s.k);
    }
    struct QR { int q; bool ok; };
    __device__ static QR qr(const GemmArgs& a, const Ctx&, int q) { return QR{q, q < a.Qdim}; }
    template <bool TAB>
    __device__ static T q_at(const GemmArgs& a, const Buf<T>& B, const Ctx& c, const QR& s, int k)
    {
        return B.at(s.ok && k < c.kend, k * a.Qdim + s.q);
    }
    __device__ static void store(const GemmArgs& a, const Ctx&, int p, int q, float acc)
    {
        const int idx = p * a.Qdim + q;
        if (a.mask) {
            const float m = a.mask_f32 ? static_cast<const float*>(a.mask)[idx]
                                       : to_f32<T>(static_cast<const T*>(a.mask)[idx]);
            if (!(m > 0.f)) acc = 0.f;
        }
        static_cast<T*>(a.out)[idx] = from_f32<T>(acc);
    }
};

// Weight gradient of one shard: p = output unit, q = input feature plus the bias column
// q = IN, k = sample in the shard.  Both operands row-fast.  blockIdx.z as for convolutions.
template <typename T> struct FcWgrad {
    typedef T TT;
    static constexpr bool P_IS_A = true;
    static constexpr bool P_ROW_FAST = true, Q_ROW_FAST = true;
    static constexpr bool KTAB = false, QTAB = false;
    struct PR { int p; bool ok; };
    __device__ static PR pr(const GemmArgs& a, const Ctx&, int p) { return PR{p, p < a.Pdim}; }
    __device__ static T p_atr(const GemmArgs& a, const Buf<T>& B, const Ctx& c, const PR& s, int k)
    {
        return B.at(s.ok && k < c.kend, (c.b0 + k) * a.Pdim + s.p);
    }
    struct QR { int q; bool ok; };
    __device__ static QR qr(const GemmArgs& a, const Ctx&, int q) { return QR{q, q < a.Qdim}; }
    template <bool TAB>
    __device__ static T q_at(const GemmArgs& a, const Buf<T>& B, const Ctx& c, const QR& s, int k)
    {
        const bool ok = s.ok && k < c.kend;
        const T v = B.at(ok && s.q < a.C, (c.b0 + k) * a.C + s.q);
        return (s.q == a.C) ? (ok ? one<T>() : zero<T>()) : v;
    }
    __device__ static void store(const GemmArgs& a, const Ctx& c, int p, int q, float acc)
    {
        float* g = static_cast<float*>(a.out) + c.r * a.out_ld;
        if (q < a.C) g[a.out_off + (long long)p * a.C + q] = acc;
        else g[a.bias_off + p] = acc;
    }
};

// ------------------------------------------------------------------------------------------
// Operand tile loaders: the four (row-fast | k-fast) x (P | Q) cases
// ------------------------------------------------------------------------------------------

// P operand, k-fast: the thread's k is fixed within a tile, rows step by 256/BK.
template <class Op, int BR, int BK, int N, bool RF, bool TAB> struct LoadP;
template <class Op, int BR, int BK, int N, bool TAB> struct LoadP<Op, BR, BK, N, false, TAB> {
    typedef typename Op::TT T;
    struct St {};
    __device__ static void init(const GemmArgs&, const Ctx&, St&, int, int) {}
    __device__ static void load(const GemmArgs& a, const Buf<T>& B, const Ctx& c, const St&,
                                int tid, int r0, int k0, T* out)
    {
        const typename Op::PK s = Op::pk(a, c, k0 + tid % BK);
        const int row = r0 + tid / BK;
#pragma unroll
        for (int i = 0; i < N; ++i) out[i] = Op::p_at(a, B, s, row + i * (256 / BK));
    }
    __device__ static int row(int tid, int i) { return tid / BK + i * (256 / BK); }
    __device__ static int kk(int tid, int) { return tid % BK; }
};
// P operand, row-fast: the thread's row is fixed for the whole kernel, k steps by 256/BR.
template <class Op, int BR, int BK, int N, bool TAB> struct LoadP<Op, BR, BK, N, true, TAB> {
    typedef typename Op::TT T;
    typedef typename Op::PR St;
    __device__ static void init(const GemmArgs& a, const Ctx& c, St& s, int tid, int r0)
    {
        s = Op::pr(a, c, r0 + tid % BR);
    }
    __device__ static void load(const GemmArgs& a, const Buf<T>& B, const Ctx& c, const St& s,
                                int tid, int, int k0, T* out)
    {
        const int k = k0 + tid / BR;
#pragma unroll
        for (int i = 0; i < N; ++i) out[i] = Op::p_atr(a, B, c, s, k + i * (256 / BR));
    }
    __device__ static int row(int tid, int) { return tid % BR; }
    __device__ static int kk(int tid, int i) { return tid / BR + i * (256 / BR); }
};

template <class Op, int BR, int BK, int N, bool RF, bool TAB> struct LoadQ;
template <class Op, int BR, int BK, int N, bool TAB> struct LoadQ<Op, BR, BK, N, false, TAB> {
    typedef typename Op::TT T;
    struct St {};
    __device__ static void init(const GemmArgs&, const Ctx&, St&, int, int) {}
    __device__ static void load(const GemmArgs& a, const Buf<T>& B, const Ctx& c, const St&,
                                int tid, int r0, int k0, T* out)
    {
        const typename Op::QK s = Op::qk(a, c, k0 + tid % BK);
        const int row = r0 + tid / BK;
#pragma unroll
        for (int i = 0; i < N; ++i)
            out[i] = Op::template q_atk<TAB>(a, B, c, s, row + i * (256 / BK), r0);
    }
    __device__ static int row(int tid, int i) { return tid / BK + i * (256 / BK); }
    __device__ static int kk(int tid, int) { return tid % BK; }
};
template <class Op, int BR, int BK, int N, bool TAB> struct LoadQ<Op, BR, BK, N, true, TAB> {
    typedef typename Op::TT T;
    typedef typename Op::QR St;
    __device__ static void init(const GemmArgs& a, const Ctx& c, St& s, int tid, int r0)
    {
        s = Op::qr(a, c, r0 + tid % BR);
    }
    __device__ static void load(const GemmArgs& a, const Buf<T>& B, const Ctx& c, const St& s,
                                int tid, int, int k0, T* out)
    {
        const int k = k0 + tid / BR;
#pragma unroll
        for (int i = 0; i < N; ++i) out[i] = Op::template q_at<TAB>(a, B, c, s, k + i * (256 / BR));
    }
    __device__ static int row(int tid, int) { return tid % BR; }
    __device__ static int kk(int tid, int i) { return tid / BR + i * (256 / BR); }
};

// ------------------------------------------------------------------------------------------
// The tiled MFMA kernel
// ------------------------------------------------------------------------------------------

template <class Op, int FP, int FQ, int BK, bool TAB>
__global__ __launch_bounds__(256) void igemm_kernel(const GemmArgs a)
{
    typedef typename Op::TT T;
    typedef Mma<T> M;
    constexpr int BP = 32 * FP, BQ = 32 * FQ;
    constexpr int VEC = M::VEC;
    constexpr int LDK = BK + VEC;  // 16 bytes of padding per row
    constexpr int NP = BP * BK / 256, NQ = BQ * BK / 256;
    static_assert(NP >= 1 && NQ >= 1 && (BP * BK) % 256 == 0 && (BQ * BK) % 256 == 0, "tile");
    static_assert(BK % M::KSTEP == 0 && 256 % BK == 0 && 256 % BP == 0 && 256 % BQ == 0, "BK");
    typedef LoadP<Op, BP, BK, NP, Op::P_ROW_FAST, TAB> LP;
    typedef LoadQ<Op, BQ, BK, NQ, Op::Q_ROW_FAST, TAB> LQ;
    // P reads tensor `a` for the weight-gradient and fully connected ops whose P side is an
    // activation, tensor `b` (the weights) for the convolution forward and data gradient.
    const Buf<T> bufP(Op::P_IS_A ? a.a : a.b, Op::P_IS_A ? a.a_bytes : a.b_bytes);
    const Buf<T> bufQ(Op::P_IS_A ? a.b : a.a, Op::P_IS_A ? a.b_bytes : a.a_bytes);

    __shared__ __attribute__((aligned(16))) T sP[BP * LDK];
    __shared__ __attribute__((aligned(16))) T sQ[BQ * LDK];
    extern __shared__ TabEnt tab[];  // sized at launch: kchunk (KTAB) or BQ (QTAB) entries

    Ctx c;
    decode_z(a, c);
    const int p0 = blockIdx.y * BP, q0 = blockIdx.x * BQ;
    const int tid = threadIdx.x;

    if constexpr (TAB && Op::KTAB) {
        for (int k = c.kbeg + tid; k < c.kbeg + a.kchunk; k += 256)
            tab[k - c.kbeg] = Op::ktab_entry(a, c, k);
        c.tab = tab;
        __syncthreads();
    }
    if constexpr (TAB && Op::QTAB) {
        if (tid < BQ) tab[tid] = Op::qtab_entry(a, q0 + tid);
        c.tab = tab;
        __syncthreads();
    }

    typename LP::St sp;
    typename LQ::St sq;
    LP::init(a, c, sp, tid, p0);
    LQ::init(a, c, sq, tid, q0);
    T rp[NP], rq[NQ];

    const int wave = tid >> 6, lane = tid & 63;
    const int wp = wave >> 1, wq = wave & 1;
    const int lr = lane & 15, lg = lane >> 4;

    f32x4 acc[FP][FQ];
#pragma unroll
    for (int i = 0; i < FP; ++i)
#pragma unroll
        for (int j = 0; j < FQ; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    int k0 = c.kbeg;
    if (k0 < c.kend) {
        LP::load(a, bufP, c, sp, tid, p0, k0, rp);
        LQ::load(a, bufQ, c, sq, tid, q0, k0, rq);
    }
    for (; k0 < c.kend; k0 += BK) {
#pragma unroll
        for (int i = 0; i < NP; ++i) sP[LP::row(tid, i) * LDK + LP::kk(tid, i)] = rp[i];
#pragma unroll
        for (int i = 0; i < NQ; ++i) sQ[LQ::row(tid, i) * LDK + LQ::kk(tid, i)] = rq[i];
        __syncthreads();
        if (k0 + BK < c.kend) {
            LP::load(a, bufP, c, sp, tid, p0, k0 + BK, rp);
            LQ::load(a, bufQ, c, sq, tid, q0, k0 + BK, rq);
        }
#pragma unroll
        for (int kc = 0; kc < BK / M::KSTEP; ++kc) {
            typename M::frag fa[FP], fb[FQ];
#pragma unroll
            for (int i = 0; i < FP; ++i)
                fa[i] = *reinterpret_cast<const typename M::frag*>(
                    &sP[(wp * 16 * FP + i * 16 + lr) * LDK + kc * M::KSTEP + lg * VEC]);
#pragma unroll
            for (int j = 0; j < FQ; ++j)
                fb[j] = *reinterpret_cast<const typename M::frag*>(
                    &sQ[(wq * 16 * FQ + j * 16 + lr) * LDK + kc * M::KSTEP + lg * VEC]);
#pragma unroll
            for (int i = 0; i < FP; ++i)
#pragma unroll
                for (int j = 0; j < FQ; ++j) M::run(acc[i][j], fa[i], fb[j]);
        }
        __syncthreads();
    }

    const bool split = a.splits > 1;
    float* part = a.partial + (long long)blockIdx.z * a.Pdim * a.Qdim;
#pragma unroll
    for (int i = 0; i < FP; ++i)
#pragma unroll
        for (int j = 0; j < FQ; ++j) {
            const int q = q0 + wq * 16 * FQ + j * 16 + lr;
            if (q >= a.Qdim) continue;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int p = p0 + wp * 16 * FP + i * 16 + lg * 4 + v;
                if (p >= a.Pdim) continue;
                if (split) part[(long long)p * a.Qdim + q] = acc[i][j][v];
                else Op::store(a, c, p, q, acc[i][j][v]);
            }
        }
}

// Second pass of a split reduction: the splits of every output are added in a fixed order and
// the operation's epilogue is applied.  A block covers 256/SL consecutive outputs of one
// (shard, group) with SL threads per output: thread l adds splits l, l+SL, l+2SL, ... in
// ascending order, then the SL partial sums are added in ascending l.  blockIdx.y = shard*G+group.
template <class Op, int SL>
__global__ __launch_bounds__(256) void split_epilogue(const GemmArgs a)
{
    constexpr int OPB = 256 / SL;
    __shared__ float sh[SL][OPB];
    const long long per = (long long)a.Pdim * a.Qdim;
    const int ol = threadIdx.x % OPB, l = threadIdx.x / OPB;
    const long long t = (long long)blockIdx.x * OPB + ol;
    const int rg = blockIdx.y;
    Ctx c;
    c.grp = rg % a.G;
    c.r = rg / a.G;
    c.split = 0; c.kbeg = 0; c.kend = a.Kdim; c.b0 = c.r * a.N; c.tab = nullptr;
    float s = 0.f;
    if (t < per) {
        const float* src = a.partial + ((long long)c.r * a.splits * a.G + c.grp) * per + t;
        for (int k = l; k < a.splits; k += SL) s += src[(long long)k * a.G * per];
    }
    sh[l][ol] = s;
    __syncthreads();
    if (l == 0 && t < per) {
        float tot = sh[0][ol];
#pragma unroll
        for (int j = 1; j < SL; ++j) tot += sh[j][ol];
        Op::store(a, c, (int)(t / a.Qdim), (int)(t % a.Qdim), tot);
    }
}

// ------------------------------------------------------------------------------------------
// Launch planning (shared by the workspace sizing and the launches)
// ------------------------------------------------------------------------------------------

GemmPlan plan_gemm(int dt, int Pdim, int Qdim, int Kdim, int zdim, bool allow_split)
{
    GemmPlan g{};
    g.FP = Pdim <= 32 ? 1 : 2;
    const long long tp = (Pdim + 32 * g.FP - 1) / (32 * g.FP);
    const long long t4 = (Qdim + 127) / 128;
    g.FQ = (t4 * tp * zdim >= 256) ? 4 : 2;
    const long long tiles = ((Qdim + 32 * g.FQ - 1) / (32 * g.FQ)) * tp * zdim;
    if (dt == DT_F32) g.BK = Kdim >= 64 ? 32 : 16;
    else g.BK = Kdim >= 128 ? 64 : 32;
    const long long ktiles = (Kdim + g.BK - 1) / g.BK;
    g.splits = 1;
    if (allow_split)
        while (tiles * g.splits < 512 && ktiles >= (long long)g.splits * 2 * 4 && g.splits < 64)
            g.splits *= 2;
    const int per = (Kdim + g.splits - 1) / g.splits;
    g.kchunk = (per + g.BK - 1) / g.BK * g.BK;
    g.splits = (Kdim + g.kchunk - 1) / g.kchunk;
    if (g.splits < 1) g.splits = 1;
    return g;
}

template <class Op, int FP, int FQ, int BK>
static hipError_t launch_tile(const GemmArgs& a, int gz, hipStream_t s)
{
    dim3 grid((a.Qdim + 32 * FQ - 1) / (32 * FQ), (a.Pdim + 32 * FP - 1) / (32 * FP), gz);
    if (grid.y > 65535u || grid.z > 65535u) return hipErrorInvalidConfiguration;
    const bool tab = Op::QTAB || (Op::KTAB && a.kchunk <= kMaxTab);
    const size_t shm = !tab ? 0 : sizeof(TabEnt) * (Op::KTAB ? a.kchunk : 32 * FQ);
    if (tab)
        hipLaunchKernelGGL((igemm_kernel<Op, FP, FQ, BK, true>), grid, dim3(256), shm, s, a);
    else
        hipLaunchKernelGGL((igemm_kernel<Op, FP, FQ, BK, false>), grid, dim3(256), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || a.splits <= 1) return e;
    const long long per = (long long)a.Pdim * a.Qdim;
    const int rg = gz / a.splits;
    if (a.splits >= 16)
        hipLaunchKernelGGL((split_epilogue<Op, 16>), dim3((unsigned)((per + 15) / 16), rg),
                           dim3(256), 0, s, a);
    else if (a.splits >= 4)
        hipLaunchKernelGGL((split_epilogue<Op, 4>), dim3((unsigned)((per + 63) / 64), rg),
                           dim3(256), 0, s, a);
    else
        hipLaunchKernelGGL((split_epilogue<Op, 1>), dim3((unsigned)((per + 255) / 256), rg),
                           dim3(256), 0, s, a);
    return hipGetLastError();
}

template <class Op, int BK>
static hipError_t launch_bk(const GemmArgs& a, const GemmPlan& g, int gz, hipStream_t s)
{
    if (g.FP == 1) {
        if (g.FQ == 4) return launch_tile<Op, 1, 4, BK>(a, gz, s);
        return launch_tile<Op, 1, 2, BK>(a, gz, s);
    }
    if (g.FQ == 4) return launch_tile<Op, 2, 4, BK>(a, gz, s);
    return launch_tile<Op, 2, 2, BK>(a, gz, s);
}

template <class Op>
static hipError_t dispatch(GemmArgs a, const GemmPlan& g, int zdim, float* partial, hipStream_t s)
{
    if (a.Pdim <= 0 || a.Qdim <= 0 || zdim <= 0) return hipSuccess;
    a.splits = g.splits;
    a.kchunk = g.kchunk;
    a.partial = partial;
    if (g.splits > 1 && !partial) return hipErrorInvalidValue;
    const int gz = zdim * g.splits;
    if constexpr (sizeof(typename Op::TT) == 4) {
        if (g.BK == 16) return launch_bk<Op, 16>(a, g, gz, s);
        return launch_bk<Op, 32>(a, g, gz, s);
    } else {
        if (g.BK == 32) return launch_bk<Op, 32>(a, g, gz, s);
        return launch_bk<Op, 64>(a, g, gz, s);
    }
}

static GemmArgs conv_args(const ConvGeom& g)
{
    GemmArgs a{};
    a.N = g.N; a.C = g.C; a.H = g.H; a.W = g.W; a.OC = g.OC; a.OH = g.OH; a.OW = g.OW;
    a.K = g.K; a.S = g.S; a.PD = g.PD; a.G = g.G;
    a.cg = g.C / g.G; a.og = g.OC / g.G; a.KK = g.K * g.K;
    a.splits = 1; a.kchunk = 0; a.R = 1;
    return a;
}

// GEMM sizes of every operation (P rows, Q columns, reduction, blockIdx.z extent before splits)
GemmDims conv_fwd_dims(const ConvGeom& g)
{
    return GemmDims{g.OC / g.G, g.N * g.OH * g.OW, (g.C / g.G) * g.K * g.K, g.G, true};
}
GemmDims conv_dgrad_dims(const ConvGeom& g)
{
    return GemmDims{g.C / g.G, g.N * g.H * g.W, (g.OC / g.G) * g.K * g.K, g.G, true};
}
GemmDims conv_wgrad_dims(const ConvGeom& g, int R)
{
    return GemmDims{g.OC / g.G, (g.C / g.G) * g.K * g.K + 1, g.N * g.OH * g.OW, g.G * R, true};
}
GemmDims conv_dgrad_col_dims(const ConvGeom& g)
{
    return GemmDims{(g.C / g.G) * g.K * g.K, g.N * g.OH * g.OW, g.OC / g.G, g.G, true};
}
size_t conv_dgrad_col_elems(const ConvGeom& g)
{
    return (size_t)g.C * g.K * g.K * (size_t)g.N * g.OH * g.OW;
}
bool conv_dgrad_use_col(const ConvGeom& g)
{
    // taps the implicit GEMM visits per useful multiply-add (stride 1: H*W / (OH*OW))
    const double waste = (double)g.H * g.W / ((double)g.OH * g.OW * g.S * g.S);
    return waste >= 1.5 && conv_dgrad_col_elems(g) * 4 <= (size_t)512 << 20;
}
GemmDims fc_fwd_dims(int B, int IN, int OUT) { return GemmDims{B, OUT, IN, 1, true}; }
GemmDims fc_dgrad_dims(int B, int IN, int OUT) { return GemmDims{B, IN, OUT, 1, true}; }
GemmDims fc_wgrad_dims(int Nb, int R, int IN, int OUT) { return GemmDims{OUT, IN + 1, Nb, R, true}; }

GemmPlan plan_for(int dt, const GemmDims& d)
{
    return plan_gemm(dt, d.P, d.Q, d.K, d.Z, d.allow_split);
}

size_t partial_elems(int dt, const GemmDims& d)
{
    const GemmPlan g = plan_for(dt, d);
    if (g.splits <= 1) return 0;
    return (size_t)g.splits * d.Z * (size_t)d.P * d.Q;
}

hipError_t conv_fwd(Dt dt, const ConvGeom& g, const void* x, const void* w, const float* bias,
                    void* y, bool y_f32, bool relu, float* partial, hipStream_t s)
{
    GemmArgs a = conv_args(g);
    a.a = x; a.b = w; a.out = y; a.bias = bias; a.relu = relu; a.out_f32 = y_f32 || dt == DT_F32;
    const unsigned es = dt == DT_F32 ? 4 : 2;
    a.a_bytes = (unsigned)((size_t)g.N * g.C * g.H * g.W * es);
    a.b_bytes = (unsigned)((size_t)g.OC * a.cg * a.KK * es);
    const GemmDims d = conv_fwd_dims(g);
    a.Pdim = d.P; a.Qdim = d.Q; a.Kdim = d.K;
    const GemmPlan p = plan_for(dt, d);
    return dt == DT_F32 ? dispatch<ConvFwd<float>>(a, p, d.Z, partial, s)
                        : dispatch<ConvFwd<bf16_t>>(a, p, d.Z, partial, s);
}

hipError_t conv_dgrad(Dt dt, const ConvGeom& g, const void* dy, const void* w, void* dx,
                      const void* mask, bool mask_f32, float* partial, hipStream_t s)
{
    GemmArgs a = conv_args(g);
    a.a = dy; a.b = w; a.out = dx; a.mask = mask; a.mask_f32 = mask_f32;
    const unsigned es = dt == DT_F32 ? 4 : 2;
    a.a_bytes = (unsigned)((size_t)g.N * g.OC * g.OH * g.OW * es);
    a.b_bytes = (unsigned)((size_t)g.OC * a.cg * a.KK * es);
    const GemmDims d = conv_dgrad_dims(g);
    a.Pdim = d.P; a.Qdim = d.Q; a.Kdim = d.K;
    const GemmPlan p = plan_for(dt, d);
    if (g.S == 1)
        return dt == DT_F32 ? dispatch<ConvDgrad<float, true>>(a, p, d.Z, partial, s)
                            : dispatch<ConvDgrad<bf16_t, true>>(a, p, d.Z, partial, s);
    return dt == DT_F32 ? dispatch<ConvDgrad<float, false>>(a, p, d.Z, partial, s)
                        : dispatch<ConvDgrad<bf16_t, false>>(a, p, d.Z, partial, s);
}

hipError_t conv_dgrad_col(Dt dt, const ConvGeom& g, const void* dy, const void* w, void* dx,
                          const void* mask, bool mask_f32, float* col, float* partial,
                          hipStream_t s)
{
    GemmArgs a = conv_args(g);
    a.a = dy; a.b = w; a.out = col;
    const unsigned es = dt == DT_F32 ? 4 : 2;
    a.a_bytes = (unsigned)((size_t)g.N * g.OC * g.OH * g.OW * es);
    a.b_bytes = (unsigned)((size_t)g.OC * a.cg * a.KK * es);
    const GemmDims d = conv_dgrad_col_dims(g);
    a.Pdim = d.P; a.Qdim = d.Q; a.Kdim = d.K;
    const GemmPlan p = plan_for(dt, d);
    hipError_t e = dt == DT_F32 ? dispatch<ConvDgradCol<float>>(a, p, d.Z, partial, s)
                                : dispatch<ConvDgradCol<bf16_t>>(a, p, d.Z, partial, s);
    if (e != hipSuccess) return e;
    GemmArgs c = conv_args(g);
    c.out = dx; c.mask = mask; c.mask_f32 = mask_f32;
    if (dt == DT_F32) launch_col2im<float>(c, col, s);
    else launch_col2im<bf16_t>(c, col, s);
    return hipGetLastError();
}

hipError_t conv_wgrad(Dt dt, const ConvGeom& g, int R, const void* x, const void* dy,
                      float* grads, long long ld, long long w_off, long long b_off,
                      float* partial, hipStream_t s)
{
    GemmArgs a = conv_args(g);
    a.a = dy; a.b = x; a.out = grads; a.out_ld = ld; a.out_off = w_off; a.bias_off = b_off;
    a.R = R;
    const unsigned es = dt == DT_F32 ? 4 : 2;
    a.a_bytes = (unsigned)((size_t)R * g.N * g.OC * g.OH * g.OW * es);
    a.b_bytes = (unsigned)((size_t)R * g.N * g.C * g.H * g.W * es);
    const GemmDims d = conv_wgrad_dims(g, R);
    a.Pdim = d.P; a.Qdim = d.Q; a.Kdim = d.K;
    const GemmPlan p = plan_for(dt, d);
    return dt == DT_F32 ? dispatch<ConvWgrad<float>>(a, p, d.Z, partial, s)
                        : dispatch<ConvWgrad<bf16_t>>(a, p, d.Z, partial, s);
}

hipError_t fc_fwd(Dt dt, int B, int IN, int OUT, const void* x, const void* w, const float* bias,
                  void* y, bool y_f32, bool relu, float* partial, hipStream_t s)
{
    GemmArgs a{};
    a.a = x; a.b = w; a.out = y; a.bias = bias; a.relu = relu; a.out_f32 = y_f32 || dt == DT_F32;
    a.N = B; a.C = IN; a.OC = OUT; a.G = 1; a.R = 1;
    const unsigned es = dt == DT_F32 ? 4 : 2;
    a.a_bytes = (unsigned)((size_t)B * IN * es);
    a.b_bytes = (unsigned)((size_t)OUT * IN * es);
    const GemmDims d = fc_fwd_dims(B, IN, OUT);
    a.Pdim = d.P; a.Qdim = d.Q; a.Kdim = d.K;
    const GemmPlan p = plan_for(dt, d);
    return dt == DT_F32 ? dispatch<FcFwd<float>>(a, p, d.Z, partial, s)
                        : dispatch<FcFwd<bf16_t>>(a, p, d.Z, partial, s);
}

hipError_t fc_dgrad(Dt dt, int B, int IN, int OUT, const void* dy, const void* w, void* dx,
                    const void* mask, bool mask_f32, float* partial, hipStream_t s)
{
    GemmArgs a{};
    a.a = dy; a.b = w; a.out = dx; a.mask = mask; a.mask_f32 = mask_f32;
    a.N = B; a.C = IN; a.OC = OUT; a.G = 1; a.R = 1;
    const unsigned es = dt == DT_F32 ? 4 : 2;
    a.a_bytes = (unsigned)((size_t)B * OUT * es);
    a.b_bytes = (unsigned)((size_t)OUT * IN * es);
    const GemmDims d = fc_dgrad_dims(B, IN, OUT);
    a.Pdim = d.P; a.Qdim = d.Q; a.Kdim = d.K;
    const GemmPlan p = plan_for(dt, d);
    return dt == DT_F32 ? dispatch<FcDgrad<float>>(a, p, d.Z, partial, s)
                        : dispatch<FcDgrad<bf16_t>>(a, p, d.Z, partial, s);
}

hipError_t fc_wgrad(Dt dt, int Nb, int R, int IN, int OUT, const void* x, const void* dy,
                    float* grads, long long ld, long long w_off, long long b_off, float* partial,
                    hipStream_t s)
{
    GemmArgs a{};
    a.a = dy; a.b = x; a.out = grads; a.out_ld = ld; a.out_off = w_off; a.bias_off = b_off;
    a.N = Nb; a.C = IN; a.OC = OUT; a.G = 1; a.R = R;
    const unsigned es = dt == DT_F32 ? 4 : 2;
    a.a_bytes = (unsigned)((size_t)R * Nb * OUT * es);
    a.b_bytes = (unsigned)((size_t)R * Nb * IN * es);
    const GemmDims d = fc_wgrad_dims(Nb, R, IN, OUT);
    a.Pdim = d.P; a.Qdim = d.Q; a.Kdim = d.K;
    const GemmPlan p = plan_for(dt, d);
    return dt == DT_F32 ? dispatch<FcWgrad<float>>(a, p, d.Z, partial, s)
                        : dispatch<FcWgrad<bf16_t>>(a, p, d.Z, partial, s);
}

}  // namespace mtx
