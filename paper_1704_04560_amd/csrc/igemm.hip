// Implicit-GEMM kernels on the gfx950 matrix cores for the convolution and fully connected
// layers: forward (+bias, +ReLU), data gradient (+ReLU mask of the layer below) and weight
// gradient (per shard, optional split of the reduction with a deterministic second pass).
//
// Every operation is written as C[p][q] = sum_k P[p][k] * Q[q][k].  An operation class
// supplies element loaders for P and Q (which gather through the convolution index map, with
// zero padding and tails returning 0) and an epilogue that scatters C into its tensor.  One
// kernel template stages BP x BK and BQ x BK tiles in LDS (k contiguous within a row, rows
// padded by 16 bytes) and runs 16x16 MFMA fragments over them:
//   fp32: v_mfma_f32_16x16x4_f32, four per 16-byte LDS read (lane group g feeds k = 4g + t
//         to the t-th instruction for both operands, so the product is unchanged);
//   bf16: v_mfma_f32_16x16x32_bf16, one per 16-byte read (8 values per lane).
// 256 threads = 4 waves in a 2 x 2 grid; a wave owns FP x FQ fragments of 16 x 16.
// MFMA output layout (16x16): lane l, register v holds row 4*(l/16) + v, column l%16, so the
// epilogue's consecutive lanes walk consecutive q (the contiguous dimension of the output).
#include "device_common.h"
#include "internal.h"

namespace mtx {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

template <typename T> struct Mma;

template <> struct Mma<float> {
    typedef f32x4 frag;
    static constexpr int VEC = 4;    // elements per 16-byte lane read
    static constexpr int KSTEP = 16; // k covered by one read across the 4 lane groups
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

// ------------------------------------------------------------------------------------------
// Operations
// ------------------------------------------------------------------------------------------

struct Ctx {
    int grp, r, split, kbeg, kend, b0;
};

// Convolution forward: p = output channel within the group, q = (image, oh, ow),
// k = (input channel within the group, u, v).
template <typename T> struct ConvFwd {
    typedef T TT;
    static constexpr bool P_ROW_FAST = false, Q_ROW_FAST = true;
    __device__ static void setup(const GemmArgs& a, Ctx& c)
    {
        c.grp = blockIdx.z; c.r = 0; c.split = 0; c.kbeg = 0; c.kend = a.Kdim; c.b0 = 0;
    }
    __device__ static T loadP(const GemmArgs& a, const Ctx& c, int p, int k)
    {
        if (p >= a.Pdim || k >= a.Kdim) return zero<T>();
        return static_cast<const T*>(a.b)[(long long)(c.grp * a.og + p) * a.Kdim + k];
    }
    __device__ static T loadQ(const GemmArgs& a, const Ctx& c, int q, int k)
    {
        if (q >= a.Qdim || k >= a.Kdim) return zero<T>();
        const int ohw = a.OH * a.OW;
        const int b = q / ohw, hw = q - b * ohw, ho = hw / a.OW, wo = hw - ho * a.OW;
        const int ci = k / a.KK, rr = k - ci * a.KK, u = rr / a.K, v = rr - u * a.K;
        const int hi = ho * a.S - a.PD + u, wi = wo * a.S - a.PD + v;
        if ((unsigned)hi >= (unsigned)a.H || (unsigned)wi >= (unsigned)a.W) return zero<T>();
        return static_cast<const T*>(a.a)[((long long)(b * a.C + c.grp * a.cg + ci) * a.H + hi) *
                                              a.W + wi];
    }
    __device__ static void store(const GemmArgs& a, const Ctx& c, int p, int q, float acc)
    {
        const int co = c.grp * a.og + p, ohw = a.OH * a.OW;
        const int b = q / ohw, hw = q - b * ohw;
        float v = acc + a.bias[co];
        if (a.relu) v = v > 0.f ? v : 0.f;
        const long long idx = ((long long)b * a.OC + co) * ohw + hw;
        if (a.out_f32) static_cast<float*>(a.out)[idx] = v;
        else static_cast<T*>(a.out)[idx] = from_f32<T>(v);
    }
};

// Convolution data gradient: p = input channel within the group, q = (image, h, w),
// k = (output channel within the group, u, v); dy is read where (h + pad - u) / stride lands
// on an output row (and likewise for columns).
template <typename T> struct ConvDgrad {
    typedef T TT;
    static constexpr bool P_ROW_FAST = false, Q_ROW_FAST = true;
    __device__ static void setup(const GemmArgs& a, Ctx& c)
    {
        c.grp = blockIdx.z; c.r = 0; c.split = 0; c.kbeg = 0; c.kend = a.Kdim; c.b0 = 0;
    }
    __device__ static T loadP(const GemmArgs& a, const Ctx& c, int p, int k)
    {
        if (p >= a.Pdim || k >= a.Kdim) return zero<T>();
        const int co = k / a.KK, rr = k - co * a.KK;
        return static_cast<const T*>(a.b)[((long long)(c.grp * a.og + co) * a.cg + p) * a.KK + rr];
    }
    __device__ static T loadQ(const GemmArgs& a, const Ctx& c, int q, int k)
    {
        if (q >= a.Qdim || k >= a.Kdim) return zero<T>();
        const int hw_in = a.H * a.W;
        const int b = q / hw_in, hw = q - b * hw_in, h = hw / a.W, w = hw - h * a.W;
        const int co = k / a.KK, rr = k - co * a.KK, u = rr / a.K, v = rr - u * a.K;
        int th = h + a.PD - u, tw = w + a.PD - v;
        if (th < 0 || tw < 0) return zero<T>();
        if (a.S > 1) {
            if (th % a.S || tw % a.S) return zero<T>();
            th /= a.S;
            tw /= a.S;
        }
        if (th >= a.OH || tw >= a.OW) return zero<T>();
        return static_cast<const T*>(a.a)[((long long)(b * a.OC + c.grp * a.og + co) * a.OH + th) *
                                              a.OW + tw];
    }
    __device__ static void store(const GemmArgs& a, const Ctx& c, int p, int q, float acc)
    {
        const int ci = c.grp * a.cg + p, hw_in = a.H * a.W;
        const int b = q / hw_in, hw = q - b * hw_in;
        const long long idx = ((long long)b * a.C + ci) * hw_in + hw;
        if (a.mask) {
            const float m = a.mask_f32 ? static_cast<const float*>(a.mask)[idx]
                                       : to_f32<T>(static_cast<const T*>(a.mask)[idx]);
            if (!(m > 0.f)) acc = 0.f;
        }
        static_cast<T*>(a.out)[idx] = from_f32<T>(acc);
    }
};

// Convolution weight gradient of one shard: p = output channel within the group,
// q = (input channel within the group, u, v), k = (image in the shard, oh, ow).
// blockIdx.z = (shard * splits + split) * G + group.
template <typename T> struct ConvWgrad {
    typedef T TT;
    static constexpr bool P_ROW_FAST = false, Q_ROW_FAST = false;
    __device__ static void setup(const GemmArgs& a, Ctx& c)
    {
        const int z = blockIdx.z;
        c.grp = z % a.G;
        const int rest = z / a.G;
        c.r = rest / a.splits;
        c.split = rest - c.r * a.splits;
        c.kbeg = c.split * a.kchunk;
        c.kend = min(a.Kdim, c.kbeg + a.kchunk);
        c.b0 = c.r * a.N;
    }
    __device__ static T loadP(const GemmArgs& a, const Ctx& c, int p, int k)
    {
        if (p >= a.Pdim || k >= a.Kdim) return zero<T>();
        const int ohw = a.OH * a.OW;
        const int b = k / ohw, hw = k - b * ohw;
        return static_cast<const T*>(a.a)[((long long)(c.b0 + b) * a.OC + c.grp * a.og + p) * ohw +
                                              hw];
    }
    __device__ static T loadQ(const GemmArgs& a, const Ctx& c, int q, int k)
    {
        if (q >= a.Qdim || k >= a.Kdim) return zero<T>();
        const int ci = q / a.KK, rr = q - ci * a.KK, u = rr / a.K, v = rr - u * a.K;
        const int ohw = a.OH * a.OW;
        const int b = k / ohw, hw = k - b * ohw, ho = hw / a.OW, wo = hw - ho * a.OW;
        const int hi = ho * a.S - a.PD + u, wi = wo * a.S - a.PD + v;
        if ((unsigned)hi >= (unsigned)a.H || (unsigned)wi >= (unsigned)a.W) return zero<T>();
        return static_cast<const T*>(a.b)[((long long)(c.b0 + b) * a.C + c.grp * a.cg + ci) *
                                              a.H * a.W + (long long)hi * a.W + wi];
    }
    __device__ static void store(const GemmArgs& a, const Ctx& c, int p, int q, float acc)
    {
        const int co = c.grp * a.og + p;
        const long long row = (long long)a.cg * a.KK;
        if (a.splits == 1)
            static_cast<float*>(a.out)[c.r * a.out_ld + a.out_off + co * row + q] = acc;
        else
            a.partial[((long long)(c.r * a.splits + c.split) * a.OC + co) * row + q] = acc;
    }
};

// Fully connected forward: p = sample, q = output unit, k = input feature.
template <typename T> struct FcFwd {
    typedef T TT;
    static constexpr bool P_ROW_FAST = false, Q_ROW_FAST = false;
    __device__ static void setup(const GemmArgs& a, Ctx& c)
    {
        c.grp = 0; c.r = 0; c.split = 0; c.kbeg = 0; c.kend = a.Kdim; c.b0 = 0;
    }
    __device__ static T loadP(const GemmArgs& a, const Ctx&, int p, int k)
    {
        if (p >= a.Pdim || k >= a.Kdim) return zero<T>();
        return static_cast<const T*>(a.a)[(long long)p * a.Kdim + k];
    }
    __device__ static T loadQ(const GemmArgs& a, const Ctx&, int q, int k)
    {
        if (q >= a.Qdim || k >= a.Kdim) return zero<T>();
        return static_cast<const T*>(a.b)[(long long)q * a.Kdim + k];
    }
    __device__ static void store(const GemmArgs& a, const Ctx&, int p, int q, float acc)
    {
        float v = acc + a.bias[q];
        if (a.relu) v = v > 0.f ? v : 0.f;
        const long long idx = (long long)p * a.Qdim + q;
        if (a.out_f32) static_cast<float*>(a.out)[idx] = v;
        else static_cast<T*>(a.out)[idx] = from_f32<T>(v);
    }
};

// Fully connected data gradient: p = sample, q = input feature, k = output unit.
template <typename T> struct FcDgrad {
    typedef T TT;
    static constexpr bool P_ROW_FAST = false, Q_ROW_FAST = true;
    __device__ static void setup(const GemmArgs& a, Ctx& c)
    {
        c.grp = 0; c.r = 0; c.split = 0; c.kbeg = 0; c.kend = a.Kdim; c.b0 = 0;
    }
    __device__ static T loadP(const GemmArgs& a, const Ctx&, int p, int k)
    {
        if (p >= a.Pdim || k >= a.Kdim) return zero<T>();
        return static_cast<const T*>(a.a)[(long long)p * a.Kdim + k];
    }
    __device__ static T loadQ(const GemmArgs& a, const Ctx&, int q, int k)
    {
        if (q >= a.Qdim || k >= a.Kdim) return zero<T>();
        return static_cast<const T*>(a.b)[(long long)k * a.Qdim + q];
    }
    __device__ static void store(const GemmArgs& a, const Ctx&, int p, int q, float acc)
    {
        const long long idx = (long long)p * a.Qdim + q;
        if (a.mask) {
            const float m = a.mask_f32 ? static_cast<const float*>(a.mask)[idx]
                                       : to_f32<T>(static_cast<const T*>(a.mask)[idx]);
            if (!(m > 0.f)) acc = 0.f;
        }
        static_cast<T*>(a.out)[idx] = from_f32<T>(acc);
    }
};

// Fully connected weight gradient of one shard: p = output unit, q = input feature,
// k = sample in the shard.  blockIdx.z = shard.
template <typename T> struct FcWgrad {
    typedef T TT;
    static constexpr bool P_ROW_FAST = true, Q_ROW_FAST = true;
    __device__ static void setup(const GemmArgs& a, Ctx& c)
    {
        c.grp = 0; c.r = blockIdx.z; c.split = 0; c.kbeg = 0; c.kend = a.Kdim; c.b0 = c.r * a.N;
    }
    __device__ static T loadP(const GemmArgs& a, const Ctx& c, int p, int k)
    {
        if (p >= a.Pdim || k >= a.Kdim) return zero<T>();
        return static_cast<const T*>(a.a)[(long long)(c.b0 + k) * a.Pdim + p];
    }
    __device__ static T loadQ(const GemmArgs& a, const Ctx& c, int q, int k)
    {
        if (q >= a.Qdim || k >= a.Kdim) return zero<T>();
        return static_cast<const T*>(a.b)[(long long)(c.b0 + k) * a.Qdim + q];
    }
    __device__ static void store(const GemmArgs& a, const Ctx& c, int p, int q, float acc)
    {
        static_cast<float*>(a.out)[c.r * a.out_ld + a.out_off + (long long)p * a.Qdim + q] = acc;
    }
};

// ------------------------------------------------------------------------------------------
// The tiled MFMA kernel
// ------------------------------------------------------------------------------------------

template <class Op, int FP, int FQ, int BK>
__global__ __launch_bounds__(256) void igemm_kernel(const GemmArgs a)
{
    typedef typename Op::TT T;
    typedef Mma<T> M;
    constexpr int BP = 32 * FP, BQ = 32 * FQ;
    constexpr int VEC = M::VEC;
    constexpr int LDK = BK + VEC;  // 16 bytes of padding per row
    constexpr int NP = BP * BK / 256, NQ = BQ * BK / 256;
    static_assert(NP >= 1 && NQ >= 1 && (BP * BK) % 256 == 0 && (BQ * BK) % 256 == 0, "tile");
    static_assert(BK % M::KSTEP == 0, "BK");

    __shared__ __attribute__((aligned(16))) T sP[BP * LDK];
    __shared__ __attribute__((aligned(16))) T sQ[BQ * LDK];

    Ctx c;
    Op::setup(a, c);
    const int p0 = blockIdx.y * BP, q0 = blockIdx.x * BQ;
    const int tid = threadIdx.x;
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
#pragma unroll
        for (int i = 0; i < NP; ++i) {
            const int e = tid + 256 * i;
            const int row = Op::P_ROW_FAST ? e % BP : e / BK, kk = Op::P_ROW_FAST ? e / BP : e % BK;
            rp[i] = Op::loadP(a, c, p0 + row, k0 + kk);
        }
#pragma unroll
        for (int i = 0; i < NQ; ++i) {
            const int e = tid + 256 * i;
            const int row = Op::Q_ROW_FAST ? e % BQ : e / BK, kk = Op::Q_ROW_FAST ? e / BQ : e % BK;
            rq[i] = Op::loadQ(a, c, q0 + row, k0 + kk);
        }
    }
    for (; k0 < c.kend; k0 += BK) {
#pragma unroll
        for (int i = 0; i < NP; ++i) {
            const int e = tid + 256 * i;
            const int row = Op::P_ROW_FAST ? e % BP : e / BK, kk = Op::P_ROW_FAST ? e / BP : e % BK;
            sP[row * LDK + kk] = rp[i];
        }
#pragma unroll
        for (int i = 0; i < NQ; ++i) {
            const int e = tid + 256 * i;
            const int row = Op::Q_ROW_FAST ? e % BQ : e / BK, kk = Op::Q_ROW_FAST ? e / BQ : e % BK;
            sQ[row * LDK + kk] = rq[i];
        }
        __syncthreads();
        const int kn = k0 + BK;
        if (kn < c.kend) {
#pragma unroll
            for (int i = 0; i < NP; ++i) {
                const int e = tid + 256 * i;
                const int row = Op::P_ROW_FAST ? e % BP : e / BK,
                          kk = Op::P_ROW_FAST ? e / BP : e % BK;
                rp[i] = Op::loadP(a, c, p0 + row, kn + kk);
            }
#pragma unroll
            for (int i = 0; i < NQ; ++i) {
                const int e = tid + 256 * i;
                const int row = Op::Q_ROW_FAST ? e % BQ : e / BK,
                          kk = Op::Q_ROW_FAST ? e / BQ : e % BK;
                rq[i] = Op::loadQ(a, c, q0 + row, kn + kk);
            }
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

#pragma unroll
    for (int i = 0; i < FP; ++i)
#pragma unroll
        for (int j = 0; j < FQ; ++j) {
            const int q = q0 + wq * 16 * FQ + j * 16 + lr;
            if (q >= a.Qdim) continue;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int p = p0 + wp * 16 * FP + i * 16 + lg * 4 + v;
                if (p < a.Pdim) Op::store(a, c, p, q, acc[i][j][v]);
            }
        }
}

// ------------------------------------------------------------------------------------------
// Launch: pick the tile shape from the problem size
// ------------------------------------------------------------------------------------------

template <class Op, int FP, int FQ>
static hipError_t launch_tile(const GemmArgs& a, int gz, hipStream_t s)
{
    constexpr int BK = sizeof(typename Op::TT) == 4 ? 16 : 32;
    dim3 grid((a.Qdim + 32 * FQ - 1) / (32 * FQ), (a.Pdim + 32 * FP - 1) / (32 * FP), gz);
    if (grid.y > 65535u || grid.z > 65535u) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL((igemm_kernel<Op, FP, FQ, BK>), grid, dim3(256), 0, s, a);
    return hipGetLastError();
}

template <class Op>
static hipError_t dispatch(const GemmArgs& a, int gz, hipStream_t s)
{
    if (a.Pdim <= 0 || a.Qdim <= 0 || gz <= 0) return hipSuccess;
    const long long q128 = (a.Qdim + 127) / 128;
    if (a.Pdim <= 32) {
        if (q128 * ((a.Pdim + 31) / 32) * gz >= 512) return launch_tile<Op, 1, 4>(a, gz, s);
        return launch_tile<Op, 1, 2>(a, gz, s);
    }
    if (q128 * ((a.Pdim + 63) / 64) * gz >= 512) return launch_tile<Op, 2, 4>(a, gz, s);
    return launch_tile<Op, 2, 2>(a, gz, s);
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

hipError_t conv_fwd(Dt dt, const ConvGeom& g, const void* x, const void* w, const float* bias,
                    void* y, bool y_f32, bool relu, hipStream_t s)
{
    GemmArgs a = conv_args(g);
    a.a = x; a.b = w; a.out = y; a.bias = bias; a.relu = relu; a.out_f32 = y_f32 || dt == DT_F32;
    a.Pdim = a.og; a.Qdim = g.N * g.OH * g.OW; a.Kdim = a.cg * a.KK;
    return dt == DT_F32 ? dispatch<ConvFwd<float>>(a, g.G, s) : dispatch<ConvFwd<bf16_t>>(a, g.G, s);
}

hipError_t conv_dgrad(Dt dt, const ConvGeom& g, const void* dy, const void* w, void* dx,
                      const void* mask, bool mask_f32, hipStream_t s)
{
    GemmArgs a = conv_args(g);
    a.a = dy; a.b = w; a.out = dx; a.mask = mask; a.mask_f32 = mask_f32;
    a.Pdim = a.cg; a.Qdim = g.N * g.H * g.W; a.Kdim = a.og * a.KK;
    return dt == DT_F32 ? dispatch<ConvDgrad<float>>(a, g.G, s)
                        : dispatch<ConvDgrad<bf16_t>>(a, g.G, s);
}

int conv_wgrad_splits(Dt, const ConvGeom& g, int R)
{
    const long long og = g.OC / g.G, cols = (long long)(g.C / g.G) * g.K * g.K;
    const long long tiles = ((og + (og <= 32 ? 31 : 63)) / (og <= 32 ? 32 : 64)) *
                            ((cols + 127) / 128) * g.G * R;
    const long long kdim = (long long)g.N * g.OH * g.OW;
    long long splits = (1024 + tiles - 1) / tiles;
    const long long max_by_k = kdim / 256;  // every split keeps at least 256 reduction steps
    if (splits > max_by_k) splits = max_by_k;
    if (splits > 64) splits = 64;
    if (splits < 1) splits = 1;
    return (int)splits;
}

size_t conv_wgrad_partial_elems(const ConvGeom& g, int R, int splits)
{
    if (splits <= 1) return 0;
    return (size_t)R * splits * g.OC * (size_t)(g.C / g.G) * g.K * g.K;
}

hipError_t conv_wgrad(Dt dt, const ConvGeom& g, int R, const void* x, const void* dy,
                      float* grads, long long ld, long long w_off, float* partial, int splits,
                      hipStream_t s)
{
    GemmArgs a = conv_args(g);
    a.a = dy; a.b = x; a.out = grads; a.partial = partial; a.out_ld = ld; a.out_off = w_off;
    a.Pdim = a.og; a.Qdim = a.cg * a.KK; a.Kdim = g.N * g.OH * g.OW;
    a.R = R; a.splits = splits < 1 ? 1 : splits;
    const int per = (a.Kdim + a.splits - 1) / a.splits;
    a.kchunk = (per + 31) / 32 * 32;
    hipError_t e = dt == DT_F32 ? dispatch<ConvWgrad<float>>(a, g.G * R * a.splits, s)
                                : dispatch<ConvWgrad<bf16_t>>(a, g.G * R * a.splits, s);
    if (e != hipSuccess || a.splits == 1) return e;
    return wgrad_reduce(R, a.splits, g.OC, a.cg * a.KK, partial, grads, ld, w_off, s);
}

hipError_t fc_fwd(Dt dt, int B, int IN, int OUT, const void* x, const void* w, const float* bias,
                  void* y, bool y_f32, bool relu, hipStream_t s)
{
    GemmArgs a{};
    a.a = x; a.b = w; a.out = y; a.bias = bias; a.relu = relu; a.out_f32 = y_f32 || dt == DT_F32;
    a.N = B; a.C = IN; a.OC = OUT; a.Pdim = B; a.Qdim = OUT; a.Kdim = IN;
    return dt == DT_F32 ? dispatch<FcFwd<float>>(a, 1, s) : dispatch<FcFwd<bf16_t>>(a, 1, s);
}

hipError_t fc_dgrad(Dt dt, int B, int IN, int OUT, const void* dy, const void* w, void* dx,
                    const void* mask, bool mask_f32, hipStream_t s)
{
    GemmArgs a{};
    a.a = dy; a.b = w; a.out = dx; a.mask = mask; a.mask_f32 = mask_f32;
    a.N = B; a.C = IN; a.OC = OUT; a.Pdim = B; a.Qdim = IN; a.Kdim = OUT;
    return dt == DT_F32 ? dispatch<FcDgrad<float>>(a, 1, s) : dispatch<FcDgrad<bf16_t>>(a, 1, s);
}

hipError_t fc_wgrad(Dt dt, int Nb, int R, int IN, int OUT, const void* x, const void* dy,
                    float* grads, long long ld, long long w_off, hipStream_t s)
{
    GemmArgs a{};
    a.a = dy; a.b = x; a.out = grads; a.out_ld = ld; a.out_off = w_off;
    a.N = Nb; a.C = IN; a.OC = OUT; a.Pdim = OUT; a.Qdim = IN; a.Kdim = Nb; a.R = R;
    return dt == DT_F32 ? dispatch<FcWgrad<float>>(a, R, s) : dispatch<FcWgrad<bf16_t>>(a, R, s);
}

}  // namespace mtx
