// Implicit-GEMM machinery on the gfx950 matrix cores, shared by the forward, data-gradient and
// weight-gradient kernel files: operand loaders, LDS tile layout, the tiled MFMA kernel, the
// split-reduction epilogue and the launch dispatch.  The operations themselves (index maps and
// epilogues) are in igemm_ops.h.
//
// Every operation is C[p][q] = sum_k P[p][k] * Q[q][k].  A block of 256 threads (4 waves in a
// 2 x 2 grid) computes a 32*FP x 32*FQ tile of C; a wave owns FP x FQ fragments of 16 x 16:
//   fp32: v_mfma_f32_16x16x4_f32, four per 16-byte LDS read (lane group g supplies
//         k = 4g + t to the t-th instruction for both operands, so the sum is unchanged);
//   bf16: v_mfma_f32_16x16x32_bf16, one per 16-byte read (8 values per lane).
// Fragment output layout: lane l, register v -> row 4*(l/16) + v, column l%16, so each lane
// ends with four consecutive rows p of one column q.
//
// Register-staged k-contiguous LDS tiles hold BR rows x BK reduction steps, rows padded by 32
// bytes, and the 16-byte granules of row r rotated by r/16.  Measured on gfx950 (LDS
// bank-conflict counters over the exact access patterns of this kernel): fragment reads run at
// the full 256 bytes per clock and 16-byte tile writes at the write rate; 16 bytes of padding
// would halve the read rate.  Direct (KD) and k-major (RT) tiles have layouts of their own,
// described with them.
//
// Operand loaders (per operand, chosen by the operation and the alignment of its tensor):
//   SK  scalar, k-fast: a thread keeps one k per tile and steps over rows;
//   SR  scalar, row-fast: a thread keeps one row for the whole kernel and loads VEC
//       consecutive k of it per pass (one 16-byte LDS store);
//   KV  16 bytes along k through registers (one LDS store per load);
//   KD  16 bytes along k straight into LDS (fp32);
//   RT  16 bytes along the rows (weight-gradient operands, whose reduction index is the
//       position), stored as loaded into a k-major tile; bf16 fragments come back through the
//       transposing LDS read, fp32 ones as four 4-byte reads.
// All global reads are raw buffer loads: the resource holds the tensor's size and the hardware
// returns 0 past it, so zero padding, tile tails and invalid rows only select an out-of-range
// offset, without branches.
//
// Reduction splits: when the output tiles alone cannot fill the GPU, the reduction is split
// over blockIdx.z; every split writes fp32 partial sums and split_epilogue adds them in a
// fixed order and applies the operation's epilogue (deterministic, no atomics).
#pragma once

#include <type_traits>

#include "device_common.h"
#include "internal.h"

namespace mtx {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));

template <typename T> struct Mma;

template <> struct Mma<float> {
    typedef f32x4 frag;
    static constexpr int VEC = 4;     // elements per 16 bytes
    static constexpr int KSTEP = 16;  // k covered by one 16-byte read across the 4 lane groups
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

// 16 bytes holding the value 1 followed by zeros (first chunk of a bias row)
template <typename T> __device__ __forceinline__ u32x4 one_chunk()
{
    if constexpr (sizeof(T) == 4) return u32x4{0x3f800000u, 0u, 0u, 0u};
    else return u32x4{0x3f80u, 0u, 0u, 0u};
}

__device__ __forceinline__ unsigned fdiv(const FastDiv& f, unsigned n)
{
    return (__umulhi(n, f.m) + n) >> f.s;
}

// ---- buffer loads -------------------------------------------------------------------------
constexpr unsigned kOOB = 0x80000000u;        // every tensor is smaller than 2 GiB
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
    // 16 bytes starting at element idx (idx is a multiple of 16 / sizeof(T))
    __device__ __forceinline__ u32x4 at16(bool ok, int idx) const
    {
        const int off = ok ? idx * (int)sizeof(T) : (int)kOOB;
        return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
    }
};

constexpr int kFar = 1 << 14;  // window coordinate that fails every bounds test

// One entry of an index table: an element offset and the two window coordinates it stands
// for (for the zero-padding test).
struct TabEnt {
    int off;
    short u, v;
};

// One 8-byte LDS read per entry.
__device__ __forceinline__ TabEnt ld_tab(const TabEnt* p)
{
    const u32x2 w = *reinterpret_cast<const u32x2*>(p);
    return TabEnt{(int)w[0], (short)(w[1] & 0xffffu), (short)(w[1] >> 16)};
}

// Window bounds test without short-circuit branches.
__device__ __forceinline__ bool inside(int h, int w, int H, int W)
{
    return ((unsigned)h < (unsigned)H) & ((unsigned)w < (unsigned)W);
}

struct Ctx {
    int grp, r, split, kbeg, kend, b0;
    const TabEnt* tab;  // LDS index table over [kbeg, kbeg + kchunk), or null
};

// Blocks are dispatched to the 8 XCDs round-robin by linear block id, and each XCD has its own
// L2.  The tile a block computes is taken from a renumbering in which every XCD owns one
// contiguous range of tiles, ordered so that neighbouring tiles read the same rows of the
// larger operand: with SHARE_Q (convolutions: the activations are the large operand) the p
// tiles of one q tile are neighbours, otherwise (fully connected: the weights) the q tiles of
// one p tile; the reduction range (blockIdx.z) varies slowest.
struct TileId {
    int bx, by, bz;
};
template <bool SHARE_Q>
__device__ __forceinline__ TileId xcd_tile()
{
    constexpr unsigned kXcd = 8;
    const unsigned nb = gridDim.x * gridDim.y * gridDim.z;
    const unsigned hw = blockIdx.x + gridDim.x * (blockIdx.y + gridDim.y * blockIdx.z);
    const unsigned q = nb / kXcd, r = nb % kXcd, x = hw % kXcd;
    const unsigned lid = x * q + min(x, r) + hw / kXcd;
    const unsigned xy = gridDim.x * gridDim.y, bz = lid / xy, l2 = lid - bz * xy;
    if (SHARE_Q) return TileId{(int)(l2 / gridDim.y), (int)(l2 % gridDim.y), (int)bz};
    return TileId{(int)(l2 % gridDim.x), (int)(l2 / gridDim.x), (int)bz};
}

__device__ __forceinline__ void decode_z(const GemmArgs& a, Ctx& c, int z)
{
    c.grp = z % a.G;
    const int rest = z / a.G;
    c.r = rest / a.splits;
    c.split = rest - c.r * a.splits;
    c.kbeg = c.split * a.kchunk;
    c.kend = min(a.Kdim, c.kbeg + a.kchunk);
    c.b0 = c.r * a.N;
    c.tab = nullptr;
}

// ---- epilogue helpers -----------------------------------------------------------------------

// Store np (<= 4) consecutive values at element idx of an fp32 tensor or of a tensor of the
// compute type; one vector store when all four are present and the launch's rows are aligned
// (vec: uniform over the launch).
template <typename T>
__device__ __forceinline__ void store_vals(void* out, bool f32, int idx, const float* v, int np,
                                           bool vec)
{
    if (f32 || sizeof(T) == 4) {
        float* o = static_cast<float*>(out) + idx;
        if (np == 4 && vec) {
            *reinterpret_cast<f32x4*>(o) = f32x4{v[0], v[1], v[2], v[3]};
        } else {
            for (int i = 0; i < np; ++i) o[i] = v[i];
        }
    } else {
        bf16_t* o = static_cast<bf16_t*>(out) + idx;
        if (np == 4 && vec) {
            const unsigned lo = (unsigned)f32_to_bf16(v[0]) | ((unsigned)f32_to_bf16(v[1]) << 16);
            const unsigned hi = (unsigned)f32_to_bf16(v[2]) | ((unsigned)f32_to_bf16(v[3]) << 16);
            *reinterpret_cast<u32x2*>(o) = u32x2{lo, hi};
        } else {
            for (int i = 0; i < np; ++i) o[i] = f32_to_bf16(v[i]);
        }
    }
}

// Zero the values whose ReLU mask (the stored output of the layer below, same index) is not
// positive.
template <typename T>
__device__ __forceinline__ void apply_mask(const GemmArgs& a, int idx, float* v, int np)
{
    if (!a.mask) return;
    float m[4] = {0.f, 0.f, 0.f, 0.f};
    if (np == 4 && a.vec_out) {
        if (a.mask_f32) {
            const f32x4 mm = *reinterpret_cast<const f32x4*>(static_cast<const float*>(a.mask) + idx);
            m[0] = mm[0]; m[1] = mm[1]; m[2] = mm[2]; m[3] = mm[3];
        } else if constexpr (sizeof(T) == 2) {
            const u32x2 w = *reinterpret_cast<const u32x2*>(static_cast<const T*>(a.mask) + idx);
            m[0] = __uint_as_float(w[0] << 16); m[1] = __uint_as_float(w[0] & 0xffff0000u);
            m[2] = __uint_as_float(w[1] << 16); m[3] = __uint_as_float(w[1] & 0xffff0000u);
        } else {
            const f32x4 mm = *reinterpret_cast<const f32x4*>(static_cast<const T*>(a.mask) + idx);
            m[0] = mm[0]; m[1] = mm[1]; m[2] = mm[2]; m[3] = mm[3];
        }
    } else {
        for (int i = 0; i < np; ++i)
            m[i] = a.mask_f32 ? static_cast<const float*>(a.mask)[idx + i]
                              : to_f32<T>(static_cast<const T*>(a.mask)[idx + i]);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
        if (!(m[i] > 0.f)) v[i] = 0.f;
}

// Bias of output rows p..p+np-1 for the operations that have one (read once per row group).
template <class Op>
__device__ __forceinline__ f32x4 row_bias(const GemmArgs& a, const Ctx& c, int p, int np)
{
    f32x4 b = {0.f, 0.f, 0.f, 0.f};
    if constexpr (Op::HAS_BIAS) {
        const float* bp = a.bias + Op::bias_index(a, c, p);
#pragma unroll
        for (int i = 0; i < 4; ++i)
            if (i < np) b[i] = bp[i];
    }
    return b;
}

// ---- LDS tile addressing --------------------------------------------------------------------
template <int BK, int VEC> struct Lds {
    static constexpr int LDK = BK + 2 * VEC;  // row stride (32 bytes of padding)
    static constexpr int NG = BK / VEC;   // 16-byte granules per row (a power of 2)
    __device__ __forceinline__ static int at(int row, int k)
    {
        const int g = ((k / VEC) + (row >> 4)) & (NG - 1);
        return row * LDK + g * VEC + (k & (VEC - 1));
    }
    // 16 bytes of row rb + lr at k = kc * ks + lg * VEC (one MFMA operand fragment)
    template <typename F, typename T>
    __device__ __forceinline__ static F frag(const T* t, int rb, int lr, int lg, int kc, int ks)
    {
        return *reinterpret_cast<const F*>(&t[at(rb + lr, kc * ks + lg * VEC)]);
    }
};

// ---- operand loaders --------------------------------------------------------------------------
enum { L_SK = 0, L_SR = 1, L_KV = 2, L_KD = 4, L_RT = 5 };

// ---- direct loads (KD): 16 bytes along k from global memory straight into LDS -----------------
// buffer_load_dwordx4 with the LDS flag: lane l of a wave writes LDS bytes [16 l, 16 l + 16) after
// the wave-uniform base in M0, so one load fills 1 KB of the tile.  The tile rows are unpadded
// (BK elements); granule g of row r sits at slot g ^ swz(r), swz(r) = (r / RW) mod NG with RW
// rows per 256 bytes, which lets the 16 rows x 4 granules of a fragment read cover distinct
// banks (measured on gfx950: 4.6 clocks per ds_read_b128 per compute unit, as for the padded
// layout, against 16.6 without the swizzle).  The lane that fills slot s of row r loads granule
// s ^ swz(r).  Loads past the tensor return zeros, as for the register loads.
template <int BK, int VEC> struct LdsD {
    static constexpr int NG = BK / VEC;
    static constexpr int RW = 16 / NG > 0 ? 16 / NG : 1;
    static constexpr int SIZE_ROWS = BK;  // elements per row
    __device__ __forceinline__ static int swz(int row) { return (row / RW) & (NG - 1); }
    __device__ __forceinline__ static int at(int row, int k)
    {
        return row * BK + (((k / VEC) ^ swz(row)) * VEC) + (k & (VEC - 1));
    }
    template <typename F, typename T>
    __device__ __forceinline__ static F frag(const T* t, int rb, int lr, int lg, int kc, int ks)
    {
        return *reinterpret_cast<const F*>(&t[at(rb + lr, kc * ks + lg * VEC)]);
    }
};

// ---- k-major tiles read with the transposing LDS load (RT, bf16) ---------------------------
// The weight-gradient operands arrive 16 bytes along the rows (8 rows at one k).  They are
// stored as loaded, T[k][row], and the MFMA fragments (8 consecutive k of one row per lane)
// come from ds_read_b64_tr_b16: within each group of 16 lanes, output lane i, element c is
// element i % 4 of the 8 bytes addressed by lane 4c + i / 4 (measured on gfx950).  So lane j of
// a group addresses rows rb + 4 (j % 4) .. + 3 at k = k0 + j / 4, and lane i receives k0 .. k0+3
// of row rb + i; a second read at k0 + 4 completes the 8 values.  The 32-byte units (16 rows) of
// k-row k sit at unit u ^ sw(k).  Two lane groups read k-rows {k0 .. k0+3, k0+8 .. k0+11}
// together; sw spreads those 8 over distinct 32-byte bank slots given how many k-rows share a
// 256-byte bank window (one for 128 rows, two for 64, four for 32).
typedef short s16x4 __attribute__((ext_vector_type(4)));
template <int BR, int BK> struct LdsT {
    static constexpr int NU = BR / 16;  // 32-byte units per k-row
    static_assert(NU == 2 || NU == 4 || NU == 8, "k-major tile rows");
    __device__ __forceinline__ static int sw(int k)
    {
        if constexpr (NU == 8) return (k & 3) | ((k >> 1) & 4);
        else if constexpr (NU == 4) return ((k >> 1) & 1) | ((k >> 2) & 2);
        else return (k >> 3) & 1;
    }
    __device__ __forceinline__ static int at(int k, int row)
    {
        return k * BR + ((((row >> 4) ^ sw(k)) << 4) | (row & 15));
    }
    template <typename F, typename T>
    __device__ __forceinline__ static F frag(const T* t, int rb, int lr, int lg, int kc, int ks)
    {
        static_assert(sizeof(T) == 2, "transposing reads are for 16-bit elements");
        const int k0 = kc * ks + lg * 8 + (lr >> 2), row = rb + 4 * (lr & 3);
        typedef __attribute__((address_space(3))) s16x4* P3;
        const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (P3)(__attribute__((address_space(3))) T*)&t[at(k0, row)]);
        const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (P3)(__attribute__((address_space(3))) T*)&t[at(k0 + 4, row)]);
        return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    }
};

// s_waitcnt immediate (gfx9 encoding) that waits until at most n vector-memory operations of the
// wave are outstanding, with no wait on the other counters
constexpr int waitcnt_vm(int n) { return (n & 15) | (7 << 4) | (15 << 8) | ((n >> 4) << 14); }

// The direct load is written as inline assembly: the compiler then does not count it, so it
// neither waits for loads into one stage before reading another nor makes every barrier wait
// for all of them; the kernels wait for them explicitly (waitcnt_vm) before the barrier that
// opens a stage.  M0 (the wave's LDS destination) is an operand of the statement.
template <typename T> struct BufD {
    u32x4 r;         // raw buffer resource: base, size in bytes, 32-bit format
    mutable T* lds;  // wave-uniform LDS destination of the next load
    __device__ __forceinline__ BufD(const void* p, unsigned bytes) : lds(nullptr)
    {
        const unsigned long long b = reinterpret_cast<unsigned long long>(p);
        r = u32x4{(unsigned)b, (unsigned)(b >> 32) & 0xffffu, bytes, kRsrcWord3};
    }
    __device__ __forceinline__ u32x4 at16(bool ok, int idx) const
    {
        const int off = ok ? idx * (int)sizeof(T) : (int)kOOB;
        const unsigned m0 = (unsigned)reinterpret_cast<unsigned long long>(
            (__attribute__((address_space(3))) T*)lds);
        asm volatile("buffer_load_dwordx4 %0, %1, 0 offen lds"
                     :
                     : "v"(off), "s"(r), "{m0}"(m0)
                     : "memory");
        return u32x4{0u, 0u, 0u, 0u};
    }
};

// LDS tile of one operand: the padded layout for register-staged loaders, the swizzled one for
// direct loads; ELEMS per stage.
template <int KIND, int BR, int BK, int VEC> struct TileOf {
    typedef Lds<BK, VEC> L;
    static constexpr int ELEMS = BR * L::LDK;
};
template <int BR, int BK, int VEC> struct TileOf<L_KD, BR, BK, VEC> {
    typedef LdsD<BK, VEC> L;
    static constexpr int ELEMS = BR * BK;
};
// fp32 k-major tile: the MFMA takes one value per lane and instruction, so a fragment is four
// 4-byte reads (k = 4 lg + t for the t-th instruction) and no transposing load is needed.  The
// 64-byte units (16 rows) of k-row k sit at unit u ^ (((k >> 2) & 3) mod units), which puts the
// four k-rows a read touches (k, k+4, k+8, k+12) on distinct bank slots for 64 rows or more.
template <int BR, int BK> struct LdsT32 {
    static constexpr int NU = BR / 16;  // 64-byte units per k-row
    static_assert(NU == 2 || NU == 4 || NU == 8, "k-major tile rows");
    __device__ __forceinline__ static int sw(int k) { return ((k >> 2) & 3) & (NU - 1); }
    __device__ __forceinline__ static int at(int k, int row)
    {
        return k * BR + ((((row >> 4) ^ sw(k)) << 4) | (row & 15));
    }
    template <typename F, typename T>
    __device__ __forceinline__ static F frag(const T* t, int rb, int lr, int lg, int kc, int ks)
    {
        static_assert(sizeof(T) == 4, "fp32 k-major tile");
        F f;
#pragma unroll
        for (int u = 0; u < 4; ++u) f[u] = t[at(kc * ks + 4 * lg + u, rb + lr)];
        return f;
    }
};

// (a 96-row tile is kept in the 128-row layout; its last 32 rows are never written or read)
template <int BR, int BK, int VEC> struct TileOf<L_RT, BR, BK, VEC> {
    static constexpr int BRL = BR == 96 ? 128 : BR;
    typedef std::conditional_t<VEC == 8, LdsT<BRL, BK>, LdsT32<BRL, BK>> L;
    static constexpr int ELEMS = BRL * BK;
};

// Per-thread loader state: the operation's type for the (side, loader) pair.
template <class Op, bool ISP, int KIND> struct LState;
template <class Op, bool ISP> struct LState<Op, ISP, L_SK> { struct type {}; };
template <class Op> struct LState<Op, true, L_SR> { typedef typename Op::PR type; };
template <class Op> struct LState<Op, true, L_KV> { typedef typename Op::PV type; };
template <class Op> struct LState<Op, true, L_KD> { typedef typename Op::PV type; };
template <class Op> struct LState<Op, false, L_KD> { typedef typename Op::QV type; };
template <class Op> struct LState<Op, true, L_RT> { typedef typename Op::PC type; };
template <class Op> struct LState<Op, false, L_RT> { typedef typename Op::QC type; };
template <class Op> struct LState<Op, false, L_SR> { typedef typename Op::QR type; };
template <class Op> struct LState<Op, false, L_KV> { typedef typename Op::QV type; };

template <class Op, bool ISP, int KIND, int BR, int BK> struct Loader;

template <class Op, bool ISP, int BR, int BK> struct Loader<Op, ISP, L_SK, BR, BK> {
    typedef typename Op::TT T;
    static constexpr int VEC = 16 / sizeof(T);
    static constexpr int RPP = 256 / BK;  // rows per pass
    static constexpr int N = (BR + RPP - 1) / RPP;
    T reg[N];
    __device__ __forceinline__ void init(const GemmArgs&, const Ctx&, int, int) {}
    __device__ __forceinline__ void load(const GemmArgs& a, const Buf<T>& B, const Ctx& c, int tid,
                                         int r0, int k0)
    {
        const int k = k0 + tid % BK;
        const int rt = tid / BK;
        if constexpr (ISP) {
            const auto s = Op::pk(a, c, k);
#pragma unroll
            for (int i = 0; i < N; ++i)
                if (RPP * N <= BR || rt + i * RPP < BR) reg[i] = Op::p_sk(a, B, c, s, r0 + rt + i * RPP);
        } else {
            const auto s = Op::qk(a, c, k);
#pragma unroll
            for (int i = 0; i < N; ++i)
                if (RPP * N <= BR || rt + i * RPP < BR) reg[i] = Op::q_sk(a, B, c, s, r0 + rt + i * RPP);
        }
    }
    __device__ __forceinline__ void stage(T* lds, int tid) const
    {
        const int kk = tid % BK, row = tid / BK;
#pragma unroll
        for (int i = 0; i < N; ++i)
            if (RPP * N <= BR || row + i * RPP < BR) lds[Lds<BK, VEC>::at(row + i * RPP, kk)] = reg[i];
    }
};

// SR: a thread keeps one row for the whole kernel and loads VEC consecutive k of it per pass
// (scalar loads; neighbouring threads read neighbouring rows, so each load instruction is
// contiguous), then stores them with one 16-byte LDS store.
template <class Op, bool ISP, int BR, int BK> struct Loader<Op, ISP, L_SR, BR, BK> {
    typedef typename Op::TT T;
    static constexpr int VEC = 16 / sizeof(T);
    static constexpr int GP = 256 / BR;   // k groups per pass
    static constexpr int KPP = GP * VEC;  // k per pass
    static constexpr int N = (BK + KPP - 1) / KPP;
    typename LState<Op, ISP, L_SR>::type s;
    T reg[N][VEC];
    __device__ __forceinline__ void init(const GemmArgs& a, const Ctx& c, int tid, int r0)
    {
        if constexpr (ISP) s = Op::pr(a, c, r0 + tid % BR);
        else s = Op::qr(a, c, r0 + tid % BR);
    }
    __device__ __forceinline__ void load(const GemmArgs& a, const Buf<T>& B, const Ctx& c, int tid,
                                         int, int k0)
    {
        const int kg = (tid / BR) * VEC;
#pragma unroll
        for (int i = 0; i < N; ++i) {
            if (!(KPP * N <= BK || kg + i * KPP < BK)) continue;  // idle beyond the tile
#pragma unroll
            for (int e = 0; e < VEC; ++e) {
                const int k = k0 + kg + i * KPP + e;
                if constexpr (ISP) reg[i][e] = Op::p_sr(a, B, c, s, k);
                else reg[i][e] = Op::q_sr(a, B, c, s, k);
            }
        }
    }
    __device__ __forceinline__ void stage(T* lds, int tid) const
    {
        const int row = tid % BR, kg = (tid / BR) * VEC;
#pragma unroll
        for (int i = 0; i < N; ++i)
            if (KPP * N <= BK || kg + i * KPP < BK)
                *reinterpret_cast<u32x4*>(&lds[Lds<BK, VEC>::at(row, kg + i * KPP)]) =
                    *reinterpret_cast<const u32x4*>(reg[i]);
    }
};

template <class Op, bool ISP, int BR, int BK> struct Loader<Op, ISP, L_KV, BR, BK> {
    typedef typename Op::TT T;
    static constexpr int VEC = 16 / sizeof(T);
    static constexpr int NG = BK / VEC;   // granules per row
    static constexpr int RPP = 256 / NG;  // rows per pass
    static constexpr int N = (BR + RPP - 1) / RPP;
    typename LState<Op, ISP, L_KV>::type s[N];
    u32x4 reg[N];
    __device__ __forceinline__ void init(const GemmArgs& a, const Ctx& c, int tid, int r0)
    {
#pragma unroll
        for (int i = 0; i < N; ++i) {
            const int row = r0 + tid / NG + i * RPP;
            if constexpr (ISP) s[i] = Op::pv(a, c, row);
            else s[i] = Op::qv(a, c, row);
        }
    }
    __device__ __forceinline__ void load(const GemmArgs& a, const Buf<T>& B, const Ctx& c, int tid,
                                         int, int k0)
    {
        const int k = k0 + (tid % NG) * VEC;
        const int rt = tid / NG;
#pragma unroll
        for (int i = 0; i < N; ++i) {
            if (!(RPP * N <= BR || rt + i * RPP < BR)) continue;
            if constexpr (ISP) reg[i] = Op::p_kv(a, B, c, s[i], k);
            else reg[i] = Op::q_kv(a, B, c, s[i], k);
        }
    }
    __device__ __forceinline__ void stage(T* lds, int tid) const
    {
        const int g = tid % NG, row = tid / NG;
#pragma unroll
        for (int i = 0; i < N; ++i)
            if (RPP * N <= BR || row + i * RPP < BR)
                *reinterpret_cast<u32x4*>(&lds[Lds<BK, VEC>::at(row + i * RPP, g * VEC)]) = reg[i];
    }
};

// RT: 16 bytes along the rows (VEC rows at one k), stored as loaded into the k-major tile.
// A tile of 96 rows has 12 row chunks: 21 k per pass, threads 252-255 idle.
template <class Op, bool ISP, int BR, int BK> struct Loader<Op, ISP, L_RT, BR, BK> {
    typedef typename Op::TT T;
    static constexpr int VEC = 16 / sizeof(T);
    static constexpr int RCH = BR / VEC;  // row chunks per tile
    static constexpr int KPP = 256 / RCH;  // k per pass
    static constexpr int N = (BK + KPP - 1) / KPP;
    static constexpr bool ALL = 256 % RCH == 0;  // every thread has a chunk
    static_assert(BR % VEC == 0 && RCH <= 256, "RT tile");
    typedef typename TileOf<L_RT, BR, BK, VEC>::L L;
    typename LState<Op, ISP, L_RT>::type s;
    u32x4 reg[N];
    __device__ __forceinline__ void init(const GemmArgs& a, const Ctx& c, int tid, int r0)
    {
        const int row0 = r0 + (tid % RCH) * VEC;
        if constexpr (ISP) s = Op::pc(a, c, row0);
        else s = Op::qc(a, c, row0);
    }
    __device__ __forceinline__ void load(const GemmArgs& a, const Buf<T>& B, const Ctx& c, int tid,
                                         int, int k0)
    {
        const int kt = tid / RCH;
        if (!ALL && kt >= KPP) return;
#pragma unroll
        for (int i = 0; i < N; ++i) {
            if (!(KPP * N <= BK || kt + i * KPP < BK)) continue;
            if constexpr (ISP) reg[i] = Op::p_rv(a, B, c, s, k0 + kt + i * KPP);
            else reg[i] = Op::q_rv(a, B, c, s, k0 + kt + i * KPP);
        }
    }
    __device__ __forceinline__ void stage(T* lds, int tid) const
    {
        const int row0 = (tid % RCH) * VEC, kt = tid / RCH;
        if (!ALL && kt >= KPP) return;
#pragma unroll
        for (int i = 0; i < N; ++i) {
            if (!(KPP * N <= BK || kt + i * KPP < BK)) continue;
            *reinterpret_cast<u32x4*>(&lds[L::at(kt + i * KPP, row0)]) = reg[i];
        }
    }
};

template <class Op, bool ISP, int BR, int BK> struct Loader<Op, ISP, L_KD, BR, BK> {
    typedef typename Op::TT T;
    static constexpr int VEC = 16 / sizeof(T);
    static constexpr int NG = BK / VEC;   // granules per row
    static constexpr int RPP = 256 / NG;  // rows per pass (four waves)
    static constexpr int RPW = 64 / NG;   // rows per wave and load
    static constexpr int N = (BR + RPP - 1) / RPP;
    typedef LdsD<BK, VEC> L;
    static_assert(BR % RPW == 0, "KD tile");
    typename LState<Op, ISP, L_KD>::type s[N];
    __device__ __forceinline__ void init(const GemmArgs& a, const Ctx& c, int tid, int r0)
    {
#pragma unroll
        for (int i = 0; i < N; ++i) {
            const int row = r0 + tid / NG + i * RPP;
            if constexpr (ISP) s[i] = Op::pv(a, c, row);
            else s[i] = Op::qv(a, c, row);
        }
    }
    // issue the loads of the tile at k0 into the LDS stage dst
    __device__ __forceinline__ void load(const GemmArgs& a, const BufD<T>& B, const Ctx& c, int tid,
                                         int wave, T* dst, int k0)
    {
        const int rt = tid / NG;  // row within a pass
#pragma unroll
        for (int i = 0; i < N; ++i) {
            if (!(RPP * N <= BR || i * RPP + wave * RPW < BR)) continue;  // wave beyond the tile
            B.lds = dst + (i * RPP + wave * RPW) * BK;
            const int k = k0 + ((tid % NG) ^ L::swz(rt + i * RPP)) * VEC;
            if constexpr (ISP) (void)Op::p_kv(a, B, c, s[i], k);
            else (void)Op::q_kv(a, B, c, s[i], k);
        }
    }
};

// ---- the tiled MFMA kernel --------------------------------------------------------------------

// An operation that declares ROW_STORE = true (with row_out / row_len) gets the staged row
// store in the epilogue of igemm_kernel.
template <class Op, class = void> struct RowStore : std::false_type {};
template <class Op>
struct RowStore<Op, std::void_t<decltype(Op::ROW_STORE)>> : std::bool_constant<Op::ROW_STORE> {};

// An operation that declares ROW_EPI = true (with out_index, rows8, out_f32, EPI_RELU, EPI_MASK)
// has output rows q contiguous along p (NHWC activations and data gradients, the col buffer):
// with the EPI template argument, igemm_kernel stages its tile and applies the epilogue to 8
// consecutive values of a row per lane (16-byte stores of bf16 rows, 8 rows x 128 bytes per
// instruction instead of 16 rows x 32 bytes).  launch_tile takes it for short reductions
// (kEpi8MaxK), where the epilogue's traffic is a large share of the launch: the bottleneck
// network's 1x1 convolutions, step 4.42 -> 4.07 ms; for the 3x3 layers of CIFAR it measured 2%
// slower, for AlexNet no different.
constexpr int kEpi8MaxK = 512;
template <class Op, class = void> struct RowEpi : std::false_type {};
template <class Op>
struct RowEpi<Op, std::void_t<decltype(Op::ROW_EPI)>> : std::bool_constant<Op::ROW_EPI> {};

// The epilogue of 8 consecutive outputs p..p+7 of row q: bias, ReLU, the mask of the layer below,
// the store -- element by element what Op::store4 does.
template <class Op>
__device__ __forceinline__ void row_epi8(const GemmArgs& a, const Ctx& c, int p, int q, f32x4 lo,
                                         f32x4 hi)
{
    typedef typename Op::TT T;
    float v[8] = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    if constexpr (Op::HAS_BIAS) {
        const float* bp = a.bias + Op::bias_index(a, c, p);
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = v[i] + bp[i];
    }
    if constexpr (Op::EPI_RELU) {
        if (a.relu)
#pragma unroll
            for (int i = 0; i < 8; ++i) v[i] = fmaxf(v[i], 0.f);
    }
    const long long idx = Op::out_index(a, c, p, q);
    if constexpr (Op::EPI_MASK) {
        if (a.mask) {
            float m[8];
            if (a.mask_f32) {
                const f32x4 m0 = *reinterpret_cast<const f32x4*>(static_cast<const float*>(a.mask) + idx);
                const f32x4 m1 = *reinterpret_cast<const f32x4*>(static_cast<const float*>(a.mask) + idx + 4);
#pragma unroll
                for (int i = 0; i < 4; ++i) { m[i] = m0[i]; m[i + 4] = m1[i]; }
            } else if constexpr (sizeof(T) == 2) {
                const u32x4 w = *reinterpret_cast<const u32x4*>(static_cast<const T*>(a.mask) + idx);
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    m[2 * i] = __uint_as_float(w[i] << 16);
                    m[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
                }
            } else {
                const f32x4 m0 = *reinterpret_cast<const f32x4*>(static_cast<const T*>(a.mask) + idx);
                const f32x4 m1 = *reinterpret_cast<const f32x4*>(static_cast<const T*>(a.mask) + idx + 4);
#pragma unroll
                for (int i = 0; i < 4; ++i) { m[i] = m0[i]; m[i + 4] = m1[i]; }
            }
#pragma unroll
            for (int i = 0; i < 8; ++i)
                if (!(m[i] > 0.f)) v[i] = 0.f;
        }
    }
    if (sizeof(T) == 4 || Op::out_f32(a)) {
        float* o = static_cast<float*>(a.out) + idx;
        *reinterpret_cast<f32x4*>(o) = f32x4{v[0], v[1], v[2], v[3]};
        *reinterpret_cast<f32x4*>(o + 4) = f32x4{v[4], v[5], v[6], v[7]};
    } else {
        u32x4 w;
#pragma unroll
        for (int i = 0; i < 4; ++i)
            w[i] = (unsigned)f32_to_bf16(v[2 * i]) | ((unsigned)f32_to_bf16(v[2 * i + 1]) << 16);
        *reinterpret_cast<u32x4*>(static_cast<bf16_t*>(a.out) + idx) = w;
    }
}

// An operation that declares INTERLEAVE = true gets the interleaved scheduling order below.
// An operation that declares DEEP_PREFETCH = true (the bf16 fully connected forward: a product
// over a long k for a few hundred output tiles, one block per compute unit, one wave per SIMD)
// keeps three k tiles of loads in flight in registers instead of one: with no other wave to
// run, a loop that issues the next tile's loads only one tile ahead waits for most of a memory
// round trip every k tile (AlexNet FC6 / FC7 / FC8 forward 43 / 33 / 17 -> 40 / 27 / 14 us).
// Not the data gradient: its 288 blocks of FC6 then need two rounds (46 -> 67 us).
template <class Op, class = void> struct DeepPrefetch : std::false_type {};
template <class Op>
struct DeepPrefetch<Op, std::void_t<decltype(Op::DEEP_PREFETCH)>> : std::bool_constant<Op::DEEP_PREFETCH> {};

template <class Op, class = void> struct Interleave : std::false_type {};
template <class Op>
struct Interleave<Op, std::void_t<decltype(Op::INTERLEAVE)>> : std::bool_constant<Op::INTERLEAVE> {};

// An operation that declares FUSE_UPDATE = true (the fully connected weight gradient fused with
// the average + update) is launched with one block per output tile for all R shards: the block
// computes and stores the shards' tiles in ascending r, keeps their running fp32 sum, and then
// averages and updates the tile's parameters itself.
template <class Op, class = void> struct FuseUpdate : std::false_type {};
template <class Op>
struct FuseUpdate<Op, std::void_t<decltype(Op::FUSE_UPDATE)>> : std::bool_constant<Op::FUSE_UPDATE> {};

// Average + update of four consecutive parameters (16-byte aligned) or of one, with the same
// arithmetic as the stand-alone average + update kernel: g = sum / R, v = mu * v + g (skipped
// for plain SGD), w = w - lr * v, each a single fp32 rounding.
__device__ __forceinline__ void fused_update4(const GemmArgs& a, long long idx, f32x4 sum)
{
    const float fr = (float)a.R;
    f32x4 g = {sum[0] / fr, sum[1] / fr, sum[2] / fr, sum[3] / fr};
    f32x4 w = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(a.upd_w + idx));
    __builtin_nontemporal_store(g, reinterpret_cast<f32x4*>(a.upd_avg + idx));
    if (a.upd_v) {
        f32x4 v = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(a.upd_v + idx));
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = fmaf(a.upd_mu, v[e], g[e]);
        __builtin_nontemporal_store(v, reinterpret_cast<f32x4*>(a.upd_v + idx));
        g = v;
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) w[e] = fmaf(-a.upd_lr, g[e], w[e]);
    __builtin_nontemporal_store(w, reinterpret_cast<f32x4*>(a.upd_w + idx));
}
__device__ __forceinline__ void fused_update1(const GemmArgs& a, long long idx, float sum)
{
    float g = sum / (float)a.R;
    a.upd_avg[idx] = g;
    if (a.upd_v) {
        const float vn = fmaf(a.upd_mu, a.upd_v[idx], g);
        a.upd_v[idx] = vn;
        g = vn;
    }
    a.upd_w[idx] = fmaf(-a.upd_lr, g, a.upd_w[idx]);
}

template <class Op, int FP, int FQ, int BK, int PK, int QK, bool SCHED = false, bool EPI = false>
__global__ __launch_bounds__(256) void igemm_kernel(const GemmArgs a)
{
    typedef typename Op::TT T;
    typedef Mma<T> M;
    constexpr int BP = 32 * FP, BQ = 32 * FQ;
    constexpr int VEC = M::VEC;
    typedef TileOf<PK, BP, BK, VEC> TP;
    typedef TileOf<QK, BQ, BK, VEC> TQ;
    typedef typename TP::L LP;
    typedef typename TQ::L LQ;
    static_assert(BK % M::KSTEP == 0 && 256 % BK == 0, "BK");
    constexpr bool FUSE = FuseUpdate<Op>::value;
    static_assert(!(FUSE && Op::TAB), "a fused update takes no index table");
    // the staged row store: output rows q contiguous along p, and 4 KB of staging per wave (the
    // operand tiles after the main loop, or, fused, a region of its own)
    constexpr bool STAGED = RowStore<Op>::value && FP == 4 && FQ == 4 &&
                            (FUSE || (TP::ELEMS * sizeof(T) >= 8192 && TQ::ELEMS * sizeof(T) >= 8192));
    constexpr bool EPI8 = EPI && RowEpi<Op>::value && FP == 4 && FQ == 4 && !FUSE &&
                          TP::ELEMS * sizeof(T) >= 8192 && TQ::ELEMS * sizeof(T) >= 8192;

    __shared__ __attribute__((aligned(16))) T sP[TP::ELEMS];
    __shared__ __attribute__((aligned(16))) T sQ[TQ::ELEMS];
    __shared__ __attribute__((aligned(16))) float stg[FUSE ? 4096 : 4];
    extern __shared__ TabEnt tab[];  // sized at launch

    const TileId tile = xcd_tile<Op::SHARE_Q>();
    const bool split = a.splits > 1;

    // products of one k tile from the operand tiles in LDS
    auto products = [&](f32x4 (&acc)[FP][FQ], int wp, int wq, int lr, int lg) {
#pragma unroll
        for (int kc = 0; kc < BK / M::KSTEP; ++kc) {
            typename M::frag fa[FP], fb[FQ];
#pragma unroll
            for (int i = 0; i < FP; ++i)
                fa[i] = LP::template frag<typename M::frag>(sP, wp * 16 * FP + i * 16, lr, lg, kc,
                                                            M::KSTEP);
#pragma unroll
            for (int j = 0; j < FQ; ++j)
                fb[j] = LQ::template frag<typename M::frag>(sQ, wq * 16 * FQ + j * 16, lr, lg, kc,
                                                            M::KSTEP);
#pragma unroll
            for (int i = 0; i < FP; ++i)
#pragma unroll
                for (int j = 0; j < FQ; ++j) M::run(acc[i][j], fa[i], fb[j]);
        }
        if constexpr (SCHED) {
            // Scheduling order: the first k chunk's fragment reads, then one fragment read of a
            // later chunk and one global load after each MFMA, so that their latencies overlap
            // the MFMAs instead of being waited for in clusters (measured: the bf16 convolution
            // weight gradients, whose operands both come through k-major tiles, run 10-25%
            // faster; forward and data-gradient kernels, and the output-bound fully connected
            // weight gradients, run slower with it).
            constexpr int NM = FP * FQ * (BK / M::KSTEP);
            __builtin_amdgcn_sched_group_barrier(0x100, FP + FQ, 0);  // LDS reads
#pragma unroll
            for (int m = 0; m < NM; ++m) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // LDS read
                __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // global load
            }
        }
    };

    // Output rows q of the operation are contiguous along p (the fully connected weight
    // gradient: one row per output unit).  A wave whose 64 p are all inside the rows stages each
    // 16-row slice of its tile in LDS (4 KB: 16 rows x 16 chunks of 16 bytes, chunk c of row r at
    // slot c ^ r) and hands it back as 4 rows x 256 contiguous bytes per instruction instead of
    // 16 rows x 64 bytes: emit(q, p, v) gets row q's 4 values from p on.
    auto staged_rows = [&](const f32x4 (&val)[FP][FQ], float* st, int pw, int q0, int wq,
                           int lane, auto&& emit) {
        const int lr = lane & 15, lg = lane >> 4;
#pragma unroll
        for (int j = 0; j < FQ; ++j) {
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
            for (int i = 0; i < FP; ++i)  // row lr, chunk i * 4 + lg
                *reinterpret_cast<f32x4*>(st + lr * 64 + (((i * 4 + lg) ^ lr) << 2)) = val[i][j];
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
            for (int it = 0; it < 4; ++it) {
                const int r = it * 4 + (lane >> 4), ch = lane & 15;
                const f32x4 v = *reinterpret_cast<const f32x4*>(st + r * 64 + ((ch ^ r) << 2));
                const int q = q0 + wq * 16 * FQ + j * 16 + r;
                if (q < a.Qdim) emit(q, pw + ch * 4, v);
            }
        }
    };

    // The same staging, read back as 8 consecutive values of a row per lane (two 16-byte
    // chunks): 8 rows x 8 lanes per pass.
    auto staged_rows8 = [&](const f32x4 (&val)[FP][FQ], float* st, int pw, int q0, int wq,
                            int lane, auto&& emit) {
        const int lr = lane & 15, lg = lane >> 4;
#pragma unroll
        for (int j = 0; j < FQ; ++j) {
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
            for (int i = 0; i < FP; ++i)  // row lr, chunk i * 4 + lg
                *reinterpret_cast<f32x4*>(st + lr * 64 + (((i * 4 + lg) ^ lr) << 2)) = val[i][j];
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
            for (int it = 0; it < 2; ++it) {
                const int r = it * 8 + (lane >> 3), c8 = lane & 7;
                const f32x4 lo = *reinterpret_cast<const f32x4*>(st + r * 64 + (((2 * c8) ^ r) << 2));
                const f32x4 hi = *reinterpret_cast<const f32x4*>(st + r * 64 + (((2 * c8 + 1) ^ r) << 2));
                const int q = q0 + wq * 16 * FQ + j * 16 + r;
                if (q < a.Qdim) emit(q, pw + c8 * 8, lo, hi);
            }
        }
    };

    // The epilogue: the staged row store (nontemporal: only the average + update at the end of
    // the step reads the rows again, and not even it when the update is fused; measured on the
    // AlexNet step: 3.57 ms with the fragment stores, 3.38 ms staged, 3.25 ms staged and
    // nontemporal), else fp32 partial sums of a split reduction, else the operation's store.
    auto store_out = [&](const Ctx& c, const f32x4 (&acc)[FP][FQ], int p0, int q0, int tid,
                         float* st) {
        const int wave = tid >> 6, lane = tid & 63;
        const int wp = wave >> 1, wq = wave & 1;
        const int lr = lane & 15, lg = lane >> 4;
        const int pw = p0 + wp * 16 * FP;
        if constexpr (STAGED) {
            if (!split && a.vec_out && pw + 16 * FP <= Op::row_len(a)) {
                staged_rows(acc, st, pw, q0, wq, lane, [&](int q, int p, f32x4 v) {
                    __builtin_nontemporal_store(v, reinterpret_cast<f32x4*>(Op::row_out(a, c, q) + p));
                });
                return;
            }
        }
        if constexpr (EPI8) {
            if (!split && Op::rows8(a) && pw + 16 * FP <= a.Pdim) {
                staged_rows8(acc, st, pw, q0, wq, lane, [&](int q, int p, f32x4 lo, f32x4 hi) {
                    row_epi8<Op>(a, c, p, q, lo, hi);
                });
                return;
            }
        }
        float* part = a.partial + (long long)tile.bz * a.Pdim * a.Qdim;
#pragma unroll
        for (int i = 0; i < FP; ++i) {
            const int p = pw + i * 16 + lg * 4;
            if (p >= a.Pdim) continue;
            const int np = min(4, a.Pdim - p);
            if (split) {
#pragma unroll
                for (int j = 0; j < FQ; ++j) {
                    const int q = q0 + wq * 16 * FQ + j * 16 + lr;
                    if (q >= a.Qdim) continue;
                    // partial sums are stored [z][q][p]
                    float* o = part + (long long)q * a.Pdim + p;
                    if (np == 4 && (a.Pdim & 3) == 0) *reinterpret_cast<f32x4*>(o) = acc[i][j];
                    else for (int v = 0; v < np; ++v) o[v] = acc[i][j][v];
                }
            } else {
                const f32x4 rb = row_bias<Op>(a, c, p, np);
#pragma unroll
                for (int j = 0; j < FQ; ++j) {
                    const int q = q0 + wq * 16 * FQ + j * 16 + lr;
                    if (q >= a.Qdim) continue;
                    // without a bias the stored value is the sum itself (no 0 added, which would
                    // turn -0 into +0: a fused update sums exactly what is stored)
                    Op::store4(a, c, p, q, Op::HAS_BIAS ? acc[i][j] + rb : acc[i][j], np);
                }
            }
        }
    };

    const Buf<T> bufP(Op::P_IS_A ? a.a : a.b, Op::P_IS_A ? a.a_bytes : a.b_bytes);
    const Buf<T> bufQ(Op::P_IS_A ? a.b : a.a, Op::P_IS_A ? a.b_bytes : a.a_bytes);
    Loader<Op, true, PK, BP, BK> lp;
    Loader<Op, false, QK, BQ, BK> lq;

    if constexpr (!FUSE) {
        Ctx c;
        decode_z(a, c, tile.bz);
        const int p0 = tile.by * BP, q0 = tile.bx * BQ;
        const int tid = threadIdx.x;
        const int wave = tid >> 6, lane = tid & 63;
        const int wp = wave >> 1, wq = wave & 1;
        const int lr = lane & 15, lg = lane >> 4;

        if constexpr (Op::TAB) {
            // entry j stands for k = kbeg + j * TS (one per 16-byte chunk for vector Q loads)
            constexpr int TS = (Op::TAB_CHUNK && QK == L_KV) ? VEC : 1;
            const int n = a.kchunk / TS;
            for (int j = tid; j < n; j += 256) tab[j] = Op::tab_entry(a, c, c.kbeg + j * TS);
            c.tab = tab;
            __syncthreads();
        }
        lp.init(a, c, tid, p0);
        lq.init(a, c, tid, q0);

        f32x4 acc[FP][FQ];
#pragma unroll
        for (int i = 0; i < FP; ++i)
#pragma unroll
            for (int j = 0; j < FQ; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

        int k0 = c.kbeg;
        if constexpr (DeepPrefetch<Op>::value) {
            // three register stages: stage i holds k tile t with t mod 3 == i; once tile t is
            // staged into LDS its registers take the loads of tile t + 3
            Loader<Op, true, PK, BP, BK> lp1, lp2;
            Loader<Op, false, QK, BQ, BK> lq1, lq2;
            lp1.init(a, c, tid, p0);
            lq1.init(a, c, tid, q0);
            lp2.init(a, c, tid, p0);
            lq2.init(a, c, tid, q0);
            auto issue = [&](auto& xp, auto& xq, int k) {
                if (k < c.kend) {
                    xp.load(a, bufP, c, tid, p0, k);
                    xq.load(a, bufQ, c, tid, q0, k);
                }
            };
            issue(lp, lq, k0);
            issue(lp1, lq1, k0 + BK);
            issue(lp2, lq2, k0 + 2 * BK);
            auto step = [&](auto& xp, auto& xq) {
                xp.stage(sP, tid);
                xq.stage(sQ, tid);
                __syncthreads();
                issue(xp, xq, k0 + 3 * BK);
                products(acc, wp, wq, lr, lg);
                __syncthreads();
                k0 += BK;
                return k0 < c.kend;
            };
            if (k0 < c.kend)
                for (;;) {
                    if (!step(lp, lq)) break;
                    if (!step(lp1, lq1)) break;
                    if (!step(lp2, lq2)) break;
                }
        } else {
            if (k0 < c.kend) {
                lp.load(a, bufP, c, tid, p0, k0);
                lq.load(a, bufQ, c, tid, q0, k0);
            }
            for (; k0 < c.kend; k0 += BK) {
                lp.stage(sP, tid);
                lq.stage(sQ, tid);
                __syncthreads();
                if (k0 + BK < c.kend) {
                    lp.load(a, bufP, c, tid, p0, k0 + BK);
                    lq.load(a, bufQ, c, tid, q0, k0 + BK);
                }
                products(acc, wp, wq, lr, lg);
                __syncthreads();
            }
        }
        // the main loop ended with a barrier, so the operand tiles are free for the staging:
        // waves 0, 1 use sP, waves 2, 3 use sQ
        float* st = nullptr;
        if constexpr (STAGED || EPI8)
            st = reinterpret_cast<float*>(wave < 2 ? static_cast<T*>(sP) : static_cast<T*>(sQ)) +
                 (wave & 1) * 1024;
        store_out(c, acc, p0, q0, tid, st);
    } else {
        // All R shards of one output tile (blockIdx.z = 0): the shards' tiles in ascending r, each
        // stored as above, their fp32 sum kept in registers, then the tile's average + update.
        // The next shard's first operand tile is loaded during the current shard's products and
        // staged into LDS before the current shard's stores are issued, so that waiting for the
        // loads never waits for the stores (loads and stores share one counter).
        Ctx c;
        decode_z(a, c, 0);
        lp.init(a, c, threadIdx.x, tile.by * BP);  // a fused operation's loader state does not
        lq.init(a, c, threadIdx.x, tile.bx * BQ);  // depend on the shard, only its loads do
        lp.load(a, bufP, c, threadIdx.x, tile.by * BP, c.kbeg);
        lq.load(a, bufQ, c, threadIdx.x, tile.bx * BQ, c.kbeg);
        lp.stage(sP, threadIdx.x);
        lq.stage(sQ, threadIdx.x);
        __syncthreads();
        f32x4 sum[FP][FQ];
        for (int rep = 0; rep < a.R; ++rep) {
            // The index arithmetic is made to depend on the shard through an opaque zero, so
            // that the compiler recomputes it per shard instead of holding every address of the
            // tile in registers across the loop (308 registers against 152).
            int oz;
            asm volatile("s_mov_b32 %0, 0" : "=s"(oz));
            const int p0 = tile.by * BP + oz, q0 = tile.bx * BQ + oz;
            const int tid = threadIdx.x + oz;
            const int wave = tid >> 6, lane = tid & 63;
            const int wp = wave >> 1, wq = wave & 1;
            const int lr = lane & 15, lg = lane >> 4;
            Ctx cn = c;
            if (rep + 1 < a.R) decode_z(a, cn, rep + 1);

            f32x4 acc[FP][FQ];
#pragma unroll
            for (int i = 0; i < FP; ++i)
#pragma unroll
                for (int j = 0; j < FQ; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
            for (int k0 = c.kbeg; k0 < c.kend; k0 += BK) {
                const bool more = k0 + BK < c.kend, next = more || rep + 1 < a.R;
                if (more) {
                    lp.load(a, bufP, c, tid, p0, k0 + BK);
                    lq.load(a, bufQ, c, tid, q0, k0 + BK);
                } else if (next) {
                    lp.load(a, bufP, cn, tid, p0, cn.kbeg);
                    lq.load(a, bufQ, cn, tid, q0, cn.kbeg);
                }
                products(acc, wp, wq, lr, lg);
                __syncthreads();
                if (next) {
                    lp.stage(sP, tid);
                    lq.stage(sQ, tid);
                    __syncthreads();
                }
            }
            store_out(c, acc, p0, q0, tid, stg + wave * 1024);
            // running sum of the stored shard values in ascending r, as the stand-alone average
            // adds the gradient rows
#pragma unroll
            for (int i = 0; i < FP; ++i)
#pragma unroll
                for (int j = 0; j < FQ; ++j) sum[i][j] = rep == 0 ? acc[i][j] : sum[i][j] + acc[i][j];
            c = cn;
        }

        // the tile's average + update: parameters out_off + q * C + p (or the bias)
        const int p0 = tile.by * BP, q0 = tile.bx * BQ;
        const int tid = threadIdx.x;
        const int wave = tid >> 6, lane = tid & 63;
        const int wp = wave >> 1, wq = wave & 1;
        const int lr = lane & 15, lg = lane >> 4;
        const int pw = p0 + wp * 16 * FP;
        if constexpr (STAGED) {
            if (a.vec_out && pw + 16 * FP <= Op::row_len(a)) {
                staged_rows(sum, stg + wave * 1024, pw, q0, wq, lane, [&](int q, int p, f32x4 v) {
                    fused_update4(a, a.out_off + (long long)q * Op::row_len(a) + p, v);
                });
                return;
            }
        }
#pragma unroll
        for (int i = 0; i < FP; ++i) {
            const int p = pw + i * 16 + lg * 4;
#pragma unroll
            for (int j = 0; j < FQ; ++j) {
                const int q = q0 + wq * 16 * FQ + j * 16 + lr;
                if (q >= a.Qdim) continue;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const long long idx = Op::param_index(a, p + e, q);
                    if (idx >= 0) fused_update1(a, idx, sum[i][j][e]);
                }
            }
        }
    }
}

// The same product with at least one operand loaded straight into LDS (KD).  Two LDS stages: the
// loads of the next k tile (direct ones into the other stage, register ones into registers,
// staged there after the products) overlap the products of this tile, and one barrier per k
// tile separates the stages.
template <class Op, int FP, int FQ, int BK, int PK, int QK>
__global__ __launch_bounds__(256) void igemm_direct_kernel(const GemmArgs a)
{
    typedef typename Op::TT T;
    typedef Mma<T> M;
    constexpr int BP = 32 * FP, BQ = 32 * FQ;
    constexpr int VEC = M::VEC;
    typedef TileOf<PK, BP, BK, VEC> TP;
    typedef TileOf<QK, BQ, BK, VEC> TQ;
    typedef typename TP::L LP;
    typedef typename TQ::L LQ;
    static_assert(BK % M::KSTEP == 0 && 256 % BK == 0, "BK");
    static_assert(PK == L_KD || QK == L_KD, "direct kernel without a direct operand");

    // one array per stage; the loop is unrolled over the two so that each step's stages are
    // known at compile time
    __shared__ __attribute__((aligned(16))) T sP0[TP::ELEMS];
    __shared__ __attribute__((aligned(16))) T sP1[TP::ELEMS];
    __shared__ __attribute__((aligned(16))) T sQ0[TQ::ELEMS];
    __shared__ __attribute__((aligned(16))) T sQ1[TQ::ELEMS];
    extern __shared__ TabEnt tab[];  // sized at launch

    const TileId tile = xcd_tile<Op::SHARE_Q>();
    Ctx c;
    decode_z(a, c, tile.bz);
    const int p0 = tile.by * BP, q0 = tile.bx * BQ;
    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;

    if constexpr (Op::TAB) {
        constexpr int TS = (Op::TAB_CHUNK && (QK == L_KV || QK == L_KD)) ? VEC : 1;
        const int n = a.kchunk / TS;
        for (int j = tid; j < n; j += 256) tab[j] = Op::tab_entry(a, c, c.kbeg + j * TS);
        c.tab = tab;
        __syncthreads();
    }

    typedef std::conditional_t<PK == L_KD, BufD<T>, Buf<T>> BPt;
    typedef std::conditional_t<QK == L_KD, BufD<T>, Buf<T>> BQt;
    const BPt bufP(Op::P_IS_A ? a.a : a.b, Op::P_IS_A ? a.a_bytes : a.b_bytes);
    const BQt bufQ(Op::P_IS_A ? a.b : a.a, Op::P_IS_A ? a.b_bytes : a.a_bytes);
    Loader<Op, true, PK, BP, BK> lp;
    Loader<Op, false, QK, BQ, BK> lq;
    lp.init(a, c, tid, p0);
    lq.init(a, c, tid, q0);

    const int wp = wave >> 1, wq = wave & 1;
    const int lr = lane & 15, lg = lane >> 4;

    f32x4 acc[FP][FQ];
#pragma unroll
    for (int i = 0; i < FP; ++i)
#pragma unroll
        for (int j = 0; j < FQ; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    // issue the loads of the tile at k into stage (dp, dq); register loaders: into registers
    auto issue = [&](T* dp, T* dq, int k) {
        if constexpr (PK == L_KD) lp.load(a, bufP, c, tid, wave, dp, k);
        else lp.load(a, bufP, c, tid, p0, k);
        if constexpr (QK == L_KD) lq.load(a, bufQ, c, tid, wave, dq, k);
        else lq.load(a, bufQ, c, tid, q0, k);
    };
    auto stage_regs = [&](T* dp, T* dq) {
        if constexpr (PK != L_KD) lp.stage(dp, tid);
        if constexpr (QK != L_KD) lq.stage(dq, tid);
    };
    // one k tile: wait until the stage (tp, tq) is complete in every wave, start the next tile
    // into (np_, nq_), multiply, then stage the next tile's register loads
    auto step = [&](const T* tp, const T* tq, T* np_, T* nq_, int k0) {
        __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));  // this wave's direct loads of the stage
        __syncthreads();
        const bool more = k0 + BK < c.kend;
        if (more) issue(np_, nq_, k0 + BK);
#pragma unroll
        for (int kc = 0; kc < BK / M::KSTEP; ++kc) {
            typename M::frag fa[FP], fb[FQ];
#pragma unroll
            for (int i = 0; i < FP; ++i)
                fa[i] = LP::template frag<typename M::frag>(tp, wp * 16 * FP + i * 16, lr, lg,
                                                            kc, M::KSTEP);
#pragma unroll
            for (int j = 0; j < FQ; ++j)
                fb[j] = LQ::template frag<typename M::frag>(tq, wq * 16 * FQ + j * 16, lr, lg,
                                                            kc, M::KSTEP);
#pragma unroll
            for (int i = 0; i < FP; ++i)
#pragma unroll
                for (int j = 0; j < FQ; ++j) M::run(acc[i][j], fa[i], fb[j]);
        }
        if (more) stage_regs(np_, nq_);
        return more;
    };

    int k0 = c.kbeg;
    if (k0 < c.kend) {
        issue(sP0, sQ0, k0);
        stage_regs(sP0, sQ0);
        // the barrier in step() follows this wave's wait for its own loads, so every stage is
        // complete in all waves before it is read
        for (;;) {
            if (!step(sP0, sQ0, sP1, sQ1, k0)) break;
            k0 += BK;
            if (!step(sP1, sQ1, sP0, sQ0, k0)) break;
            k0 += BK;
        }
    }

    const bool split = a.splits > 1;
    float* part = a.partial + (long long)tile.bz * a.Pdim * a.Qdim;
#pragma unroll
    for (int i = 0; i < FP; ++i) {
        const int p = p0 + wp * 16 * FP + i * 16 + lg * 4;
        if (p >= a.Pdim) continue;
        const int np = min(4, a.Pdim - p);
        if (split) {
#pragma unroll
            for (int j = 0; j < FQ; ++j) {
                const int q = q0 + wq * 16 * FQ + j * 16 + lr;
                if (q >= a.Qdim) continue;
                float* o = part + (long long)q * a.Pdim + p;
                if (np == 4 && (a.Pdim & 3) == 0) *reinterpret_cast<f32x4*>(o) = acc[i][j];
                else for (int v = 0; v < np; ++v) o[v] = acc[i][j][v];
            }
        } else {
            const f32x4 rb = row_bias<Op>(a, c, p, np);
#pragma unroll
            for (int j = 0; j < FQ; ++j) {
                const int q = q0 + wq * 16 * FQ + j * 16 + lr;
                if (q >= a.Qdim) continue;
                Op::store4(a, c, p, q, acc[i][j] + rb, np);
            }
        }
    }
}

// Second pass of a split reduction.  A block covers OPB = 256/SL consecutive groups of V
// outputs t = q * Pdim + p of one (shard, group) with SL threads per group: thread l adds splits
// l, l + SL, ... in ascending order, then the SL partial sums are added in ascending l.  V = 4
// (Pdim % 4 == 0): four consecutive outputs of one row q per group, 16-byte loads and the
// operation's 4-wide store (the same sums as V = 1; AlexNet conv1's 48-split weight-gradient
// reduction 32.6 -> 18.5 us).  blockIdx.y = shard * G + group.
template <class Op, int SL, int V = 1>
__global__ __launch_bounds__(256) void split_epilogue(const GemmArgs a)
{
    static_assert(V == 1 || V == 4, "outputs per group");
    typedef std::conditional_t<V == 4, f32x4, float> Acc;
    constexpr int OPB = 256 / SL;
    __shared__ Acc sh[SL][OPB];
    const long long per = (long long)a.Pdim * a.Qdim;
    const int ol = threadIdx.x % OPB, l = threadIdx.x / OPB;
    const long long t = ((long long)blockIdx.x * OPB + ol) * V;
    const int rg = blockIdx.y;
    Ctx c;
    c.grp = rg % a.G;
    c.r = rg / a.G;
    c.split = 0;
    c.kbeg = 0;
    c.kend = a.Kdim;
    c.b0 = c.r * a.N;
    c.tab = nullptr;
    Acc s = Acc{};
    if (t < per) {
        const float* src = a.partial + ((long long)c.r * a.splits * a.G + c.grp) * per + t;
        for (int k = l; k < a.splits; k += SL)
            s += *reinterpret_cast<const Acc*>(src + (long long)k * a.G * per);
    }
    sh[l][ol] = s;
    __syncthreads();
    if (l == 0 && t < per) {
        Acc tot = sh[0][ol];
#pragma unroll
        for (int j = 1; j < SL; ++j) tot += sh[j][ol];
        const int q = (int)(t / a.Pdim), p = (int)(t - (long long)q * a.Pdim);
        if constexpr (V == 4)
            Op::store4(a, c, p, q, Op::HAS_BIAS ? tot + row_bias<Op>(a, c, p, 4) : tot, 4);
        else
            Op::store4(a, c, p, q, f32x4{tot + row_bias<Op>(a, c, p, 1)[0], 0.f, 0.f, 0.f}, 1);
    }
}

// The same second pass for fewer than 16 splits and Pdim % 4 == 0: a thread adds the splits of
// four consecutive outputs t .. t+3 (one row q, rows p .. p+3) in ascending split order with
// 16-byte loads and hands them to the operation's 4-wide store, as the main kernel's epilogue
// does (one output per thread with 4-byte loads moved AlexNet's fully connected partial sums at
// about a fifth of the HBM rate).
template <class Op>
__global__ __launch_bounds__(256) void split_epilogue4(const GemmArgs a)
{
    const long long per = (long long)a.Pdim * a.Qdim;
    const long long t = ((long long)blockIdx.x * 256 + threadIdx.x) * 4;
    if (t >= per) return;
    Ctx c;
    c.grp = blockIdx.y % a.G;
    c.r = blockIdx.y / a.G;
    c.split = 0;
    c.kbeg = 0;
    c.kend = a.Kdim;
    c.b0 = c.r * a.N;
    c.tab = nullptr;
    const float* src = a.partial + ((long long)c.r * a.splits * a.G + c.grp) * per + t;
    const long long zs = (long long)a.G * per;
    f32x4 sum = *reinterpret_cast<const f32x4*>(src);
#pragma unroll 4
    for (int k = 1; k < a.splits; ++k) sum += *reinterpret_cast<const f32x4*>(src + k * zs);
    const int q = (int)(t / a.Pdim), p = (int)(t - (long long)q * a.Pdim);
    Op::store4(a, c, p, q, Op::HAS_BIAS ? sum + row_bias<Op>(a, c, p, 4) : sum, 4);
}

// ---- launch ---------------------------------------------------------------------------------
template <class Op, int FP, int FQ, int BK, int PK, int QK>
static hipError_t launch_tile(const GemmArgs& a, int gz, hipStream_t s)
{
    typedef typename Op::TT T;
    constexpr int VEC = 16 / sizeof(T);
    if (a.kchunk % BK != 0) return hipErrorInvalidValue;  // plan and kernel disagree
    dim3 grid((a.Qdim + 32 * FQ - 1) / (32 * FQ), (a.Pdim + 32 * FP - 1) / (32 * FP), gz);
    if (grid.y > 65535u || grid.z > 65535u) return hipErrorInvalidConfiguration;
    size_t shm = 0;
    if constexpr (Op::TAB) {
        const int ts = (Op::TAB_CHUNK && (QK == L_KV || QK == L_KD)) ? VEC : 1;
        const int n = a.kchunk / ts;
        if (n > kMaxTab) return hipErrorInvalidValue;  // the plan keeps chunks within the table
        shm = sizeof(TabEnt) * (size_t)n;
    }
    if constexpr (PK == L_KD || QK == L_KD) {
        note_gemm(FP, FQ, BK, a.splits, kGemmDirectLds);
        hipLaunchKernelGGL((igemm_direct_kernel<Op, FP, FQ, BK, PK, QK>), grid, dim3(256), shm, s,
                           a);
    } else if constexpr (Interleave<Op>::value && sizeof(typename Op::TT) == 2) {
        note_gemm(FP, FQ, BK, a.splits, kGemmInterleaved);
        hipLaunchKernelGGL((igemm_kernel<Op, FP, FQ, BK, PK, QK, true>), grid, dim3(256), shm, s,
                           a);
    } else {
        note_gemm(FP, FQ, BK, a.splits, FuseUpdate<Op>::value ? kGemmFusedUpdate : 0);
        constexpr bool EPI_OK = RowEpi<Op>::value && FP == 4 && FQ == 4 && !FuseUpdate<Op>::value;
        if constexpr (EPI_OK) {
            if (a.Kdim <= kEpi8MaxK && a.splits <= 1) {
                hipLaunchKernelGGL((igemm_kernel<Op, FP, FQ, BK, PK, QK, false, true>), grid,
                                   dim3(256), shm, s, a);
                return hipGetLastError();
            }
        }
        hipLaunchKernelGGL((igemm_kernel<Op, FP, FQ, BK, PK, QK>), grid, dim3(256), shm, s, a);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || a.splits <= 1) return e;
    timing_split(s, "reduce");
    const long long per = (long long)a.Pdim * a.Qdim;
    const int rg = gz / a.splits;
    if (a.splits < 16 && a.Pdim % 4 == 0)
        hipLaunchKernelGGL((split_epilogue4<Op>), dim3((unsigned)((per / 4 + 255) / 256), rg),
                           dim3(256), 0, s, a);
    else if (a.splits >= 16 && a.Pdim % 4 == 0)
        hipLaunchKernelGGL((split_epilogue<Op, 16, 4>), dim3((unsigned)((per / 4 + 15) / 16), rg),
                           dim3(256), 0, s, a);
    else if (a.splits >= 16)
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

// Tile shapes (FP, FQ) in {(1,2), (1,4), (2,2), (2,4), (3,4), (4,4)}, k tile 32 or 64; the
// 96-row tile only for bf16 with the P operand loaded along k, or loaded 16 bytes along the rows
// when P is at most 96, else the 128-row tile (the plan's splits and chunks hold for either).
// With rows loaded along the rows the 96-row tile takes fewer products per transposing read
// than the 128-row one: measured on AlexNet's weight gradients, it pays where it replaces two
// 64-row tiles (conv1, 96 channels: 218 -> 179 us) and not where it replaces a 128-row tile of
// which a quarter is padding (the 192-channel groups of conv4: 114 -> 123 us).
template <class Op, int BK, int PK, int QK>
static hipError_t launch_shape_bk(const GemmArgs& a, const GemmPlan& g, int gz, hipStream_t s)
{
    if constexpr (sizeof(typename Op::TT) == 2 && (PK == L_KV || PK == L_SK || PK == L_RT))
        if (g.FP == 3 && (PK != L_RT || a.Pdim <= 96))
            return launch_tile<Op, 3, 4, BK, PK, QK>(a, gz, s);
    if (g.FP == 1) {
        if (g.FQ == 4) return launch_tile<Op, 1, 4, BK, PK, QK>(a, gz, s);
        return launch_tile<Op, 1, 2, BK, PK, QK>(a, gz, s);
    }
    if (g.FP == 2) {
        if (g.FQ == 4) return launch_tile<Op, 2, 4, BK, PK, QK>(a, gz, s);
        return launch_tile<Op, 2, 2, BK, PK, QK>(a, gz, s);
    }
    return launch_tile<Op, 4, 4, BK, PK, QK>(a, gz, s);
}

// Runs operation Op with loaders (PK, QK) under plan g; zdim = blocks along z before splits.
template <class Op, int PK, int QK>
static hipError_t run_gemm(GemmArgs a, const GemmPlan& g, int zdim, float* partial,
                           hipStream_t s)
{
    if (a.Pdim <= 0 || a.Qdim <= 0 || zdim <= 0) return hipSuccess;
    a.splits = g.splits;
    a.kchunk = g.kchunk;
    a.partial = partial;
    if (g.splits > 1 && !partial) return hipErrorInvalidValue;
    const int gz = zdim * g.splits;
    if (g.BK == 32) return launch_shape_bk<Op, 32, PK, QK>(a, g, gz, s);
    if (g.BK == 64) return launch_shape_bk<Op, 64, PK, QK>(a, g, gz, s);
    return hipErrorInvalidValue;
}

}  // namespace mtx
