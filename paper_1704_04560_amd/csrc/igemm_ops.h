// The operations of the implicit GEMM (see igemm.h): for each, the index maps of its two
// operands under every loader it supports, its LDS index table and its epilogue.
//
// Interface of an operation Op (only the members its loaders use need to exist):
//   TT                compute type; P_IS_A: P reads tensor a (else tensor b, Q the other)
//   SHARE_Q           neighbouring tiles share q (see xcd_tile)
//   TAB, TAB_CHUNK    an LDS table over the block's k range exists; for 16-byte Q loads it
//                     has one entry per chunk; tab_entry(a, c, k) builds an entry
//   pk/p_sk           SK loader on P: state for column k, element of row p
//   pr/p_sr           SR loader on P: state for row p, element at k
//   pv/p_kv           KV and KD loaders on P: state for row p, 16 bytes at k (B.at16 on the
//                     buffer given: a register load, or a load straight into LDS)
//   pc/p_rv           RT loader on P: state for rows p0..p0+VEC-1, 16 bytes at k
//   qk/q_sk, qr/q_sr, qv/q_kv, qc/q_rv   the same for Q
//   store4(a, c, p, q, acc, np)   epilogue for rows p..p+np-1 of column q
//   INTERLEAVE        (optional) schedule fragment reads and loads between the MFMAs
#pragma once

#include "igemm.h"

namespace mtx {

struct RowOk {
    int off;
    bool ok;
};

// Host: the convolution fields of GemmArgs, with the divisors the index maps use.
static inline GemmArgs conv_args(const ConvGeom& g)
{
    GemmArgs a{};
    a.N = g.N; a.C = g.C; a.H = g.H; a.W = g.W; a.OC = g.OC; a.OH = g.OH; a.OW = g.OW;
    a.K = g.K; a.S = g.S; a.PD = g.PD; a.G = g.G;
    a.cg = g.C / g.G; a.og = g.OC / g.G; a.KK = g.K * g.K;
    a.splits = 1; a.kchunk = 0; a.R = 1; a.perm_c = 1; a.perm_hw = 1;
    a.fd_ohw = make_fastdiv((unsigned)(g.OH * g.OW));
    a.fd_ow = make_fastdiv((unsigned)g.OW);
    a.fd_hw = make_fastdiv((unsigned)(g.H * g.W));
    a.fd_w = make_fastdiv((unsigned)g.W);
    a.fd_c = make_fastdiv((unsigned)g.C);
    a.fd_kcg = make_fastdiv((unsigned)(g.K * a.cg));
    a.fd_cg = make_fastdiv((unsigned)a.cg);
    a.fd_kog = make_fastdiv((unsigned)(g.K * a.og));
    a.fd_og = make_fastdiv((unsigned)a.og);
    a.fd_run = make_fastdiv(1u);
    return a;
}

// ------------------------------------------------------------------------------------------
// Convolution forward (eq. 1 of a convolution layer, all R shards at once):
// p = output channel in the group, q = output position (n, oh, ow), k = (u, v, ci) with ci
// innermost.  P = Wf (tensor b), Q = input patches of x (tensor a, NHWC).
// ------------------------------------------------------------------------------------------
template <typename T> struct ConvFwd {
    typedef T TT;
    static constexpr bool P_IS_A = false;
    static constexpr bool SHARE_Q = true;
    static constexpr bool TAB = true, TAB_CHUNK = true;
    __device__ static TabEnt tab_entry(const GemmArgs& a, const Ctx& c, int k)
    {
        if (k >= c.kend) return TabEnt{0, (short)kFar, (short)kFar};
        const int u = (int)fdiv(a.fd_kcg, (unsigned)k), rem = k - u * a.K * a.cg;
        const int v = (int)fdiv(a.fd_cg, (unsigned)rem), ci = rem - v * a.cg;
        return TabEnt{(u * a.W + v) * a.C + ci, (short)u, (short)v};
    }
    // P: Wf[(g*og + p) * Kdim + k]
    struct PK { int base; bool ok; };
    __device__ static PK pk(const GemmArgs& a, const Ctx& c, int k)
    {
        return PK{c.grp * a.og * a.Kdim + k, k < c.kend};
    }
    __device__ static T p_sk(const GemmArgs& a, const Buf<T>& B, const Ctx&, const PK& s, int p)
    {
        return B.at(s.ok & (p < a.Pdim), s.base + p * a.Kdim);
    }
    typedef RowOk PV;
    __device__ static PV pv(const GemmArgs& a, const Ctx& c, int p)
    {
        return PV{(c.grp * a.og + p) * a.Kdim, p < a.Pdim};
    }
    template <class BT>
    __device__ static u32x4 p_kv(const GemmArgs&, const BT& B, const Ctx& c, const PV& s, int k)
    {
        return B.at16(s.ok & (k < c.kend), s.off + k);
    }
    // Q: x[n][oh*S - PD + u][ow*S - PD + v][g*cg + ci]
    struct QR { int base, h0, w0; };
    __device__ static QR qr(const GemmArgs& a, const Ctx& c, int q)
    {
        const bool ok = q < a.Qdim;
        const unsigned qq = ok ? q : 0;
        const unsigned b = fdiv(a.fd_ohw, qq), hw = qq - b * (unsigned)(a.OH * a.OW);
        const unsigned oh = fdiv(a.fd_ow, hw), ow = hw - oh * (unsigned)a.OW;
        QR s;
        const int h0 = (int)oh * a.S - a.PD;
        s.w0 = (int)ow * a.S - a.PD;
        s.base = (((int)b * a.H + h0) * a.W + s.w0) * a.C + c.grp * a.cg;
        s.h0 = ok ? h0 : -kFar;  // an invalid row fails every bounds test
        return s;
    }
    __device__ static T q_sr(const GemmArgs& a, const Buf<T>& B, const Ctx& c, const QR& s, int k)
    {
        const TabEnt e = ld_tab(c.tab + (k - c.kbeg));
        const int hi = s.h0 + e.u, wi = s.w0 + e.v;
        return B.at(inside(hi, wi, a.H, a.W), s.base + e.off);
    }
    typedef QR QV;
    __device__ static QV qv(const GemmArgs& a, const Ctx& c, int q) { return qr(a, c, q); }
    template <class BT>
    __device__ static u32x4 q_kv(const GemmArgs& a, const BT& B, const Ctx& c, const QV& s, int k)
    {
        const TabEnt e = ld_tab(c.tab + (k - c.kbeg) / (16 / (int)sizeof(T)));
        const int hi = s.h0 + e.u, wi = s.w0 + e.v;
        return B.at16(inside(hi, wi, a.H, a.W), s.base + e.off);
    }
    static constexpr bool HAS_BIAS = true;
    __device__ static int bias_index(const GemmArgs& a, const Ctx& c, int p) { return c.grp * a.og + p; }
    // y[q][g*og + p] = acc (bias included), ReLU
    __device__ static void store4(const GemmArgs& a, const Ctx& c, int p, int q, f32x4 acc, int np)
    {
        const int co = c.grp * a.og + p;
        float v[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = a.relu ? fmaxf(acc[i], 0.f) : acc[i];
        store_vals<T>(a.out, a.out_f32, q * a.OC + co, v, np, a.vec_out);
    }
    static constexpr bool ROW_EPI = true, EPI_RELU = true, EPI_MASK = false;
    __device__ static long long out_index(const GemmArgs& a, const Ctx& c, int p, int q)
    {
        return (long long)q * a.OC + c.grp * a.og + p;
    }
    __device__ static bool rows8(const GemmArgs& a) { return a.OC % 8 == 0 && a.og % 8 == 0; }
    __device__ static bool out_f32(const GemmArgs& a) { return a.out_f32; }
};

// ------------------------------------------------------------------------------------------
// Convolution data gradient (eq. 2, the error propagated to the layer below):
// p = input channel in the group, q = input position (n, h, w), k = (u, v, co) with co
// innermost; dy at (h + PD - u, w + PD - v) / stride contributes where that is an integer
// position inside dy.  P = Wd (tensor b), Q = dy (tensor a, NHWC).
// STRIDE1: the dy offset of every k comes from the table; otherwise it is decoded per element.
// ------------------------------------------------------------------------------------------
template <typename T, bool STRIDE1> struct ConvDgrad {
    typedef T TT;
    static constexpr bool P_IS_A = false;
    static constexpr bool SHARE_Q = true;
    static constexpr bool HAS_BIAS = false;
    static constexpr bool TAB = STRIDE1, TAB_CHUNK = true;
    __device__ static TabEnt tab_entry(const GemmArgs& a, const Ctx& c, int k)
    {
        if (k >= c.kend) return TabEnt{0, (short)-kFar, (short)-kFar};
        const int u = (int)fdiv(a.fd_kog, (unsigned)k), rem = k - u * a.K * a.og;
        const int v = (int)fdiv(a.fd_og, (unsigned)rem), co = rem - v * a.og;
        return TabEnt{-(u * a.OW + v) * a.OC + co, (short)u, (short)v};
    }
    // P: Wd[(g*cg + p) * Kdim + k]
    struct PK { int base; bool ok; };
    __device__ static PK pk(const GemmArgs& a, const Ctx& c, int k)
    {
        return PK{c.grp * a.cg * a.Kdim + k, k < c.kend};
    }
    __device__ static T p_sk(const GemmArgs& a, const Buf<T>& B, const Ctx&, const PK& s, int p)
    {
        return B.at(s.ok & (p < a.Pdim), s.base + p * a.Kdim);
    }
    typedef RowOk PV;
    __device__ static PV pv(const GemmArgs& a, const Ctx& c, int p)
    {
        return PV{(c.grp * a.cg + p) * a.Kdim, p < a.Pdim};
    }
    template <class BT>
    __device__ static u32x4 p_kv(const GemmArgs&, const BT& B, const Ctx& c, const PV& s, int k)
    {
        return B.at16(s.ok & (k < c.kend), s.off + k);
    }
    // Q: dy
    struct QR { int base, hp, wp, b; };
    __device__ static QR qr(const GemmArgs& a, const Ctx& c, int q)
    {
        const bool ok = q < a.Qdim;
        const unsigned qq = ok ? q : 0;
        const unsigned b = fdiv(a.fd_hw, qq), hw = qq - b * (unsigned)(a.H * a.W);
        const unsigned h = fdiv(a.fd_w, hw), w = hw - h * (unsigned)a.W;
        QR s;
        const int hp = (int)h + a.PD;
        s.wp = (int)w + a.PD;
        s.b = (int)b;
        s.base = STRIDE1 ? (((int)b * a.OH + hp) * a.OW + s.wp) * a.OC + c.grp * a.og : 0;
        s.hp = ok ? hp : -kFar;  // an invalid row fails every bounds test
        return s;
    }
    __device__ static T q_sr(const GemmArgs& a, const Buf<T>& B, const Ctx& c, const QR& s, int k)
    {
        if constexpr (STRIDE1) {
            const TabEnt e = ld_tab(c.tab + (k - c.kbeg));
            const int th = s.hp - e.u, tw = s.wp - e.v;
            return B.at(inside(th, tw, a.OH, a.OW), s.base + e.off);
        } else {
            const bool kok = k < c.kend;
            const int kk = kok ? k : 0;
            const int kc = a.K * a.og;
            const int u = kk / kc, rem = kk - u * kc, v = rem / a.og, co = rem - v * a.og;
            const int th = s.hp - u, tw = s.wp - v;
            const int oh = th / a.S, ow = tw / a.S;
            const bool ok = kok && th >= 0 && tw >= 0 && oh * a.S == th && ow * a.S == tw &&
                            oh < a.OH && ow < a.OW;
            return B.at(ok, ((s.b * a.OH + oh) * a.OW + ow) * a.OC + c.grp * a.og + co);
        }
    }
    typedef QR QV;
    __device__ static QV qv(const GemmArgs& a, const Ctx& c, int q) { return qr(a, c, q); }
    template <class BT>
    __device__ static u32x4 q_kv(const GemmArgs& a, const BT& B, const Ctx& c, const QV& s, int k)
    {
        const TabEnt e = ld_tab(c.tab + (k - c.kbeg) / (16 / (int)sizeof(T)));
        const int th = s.hp - e.u, tw = s.wp - e.v;
        return B.at16(inside(th, tw, a.OH, a.OW), s.base + e.off);
    }
    // dx[q][g*cg + p] = acc, times the ReLU mask of the layer below
    __device__ static void store4(const GemmArgs& a, const Ctx& c, int p, int q, f32x4 acc, int np)
    {
        const int idx = q * a.C + c.grp * a.cg + p;
        float v[4] = {acc[0], acc[1], acc[2], acc[3]};
        apply_mask<T>(a, idx, v, np);
        store_vals<T>(a.out, false, idx, v, np, a.vec_out);
    }
    static constexpr bool ROW_EPI = true, EPI_RELU = false, EPI_MASK = true;
    __device__ static long long out_index(const GemmArgs& a, const Ctx& c, int p, int q)
    {
        return (long long)q * a.C + c.grp * a.cg + p;
    }
    __device__ static bool rows8(const GemmArgs& a) { return a.C % 8 == 0 && a.cg % 8 == 0; }
    __device__ static bool out_f32(const GemmArgs&) { return false; }
};

// ------------------------------------------------------------------------------------------
// Convolution data gradient in two passes, for convolutions whose implicit data-gradient GEMM
// would spend much of its reduction on taps outside dy (unpadded convolutions):
//   col[g][q][p] = sum_co Wc[g][p][co] * dy[q][g*og + co],  p = (u, v, ci), q = (n, oh, ow)
// (an exact GEMM, k = co), then col2im_kernel gathers dx from col (fp32).
// ------------------------------------------------------------------------------------------
template <typename T> struct ConvDgradCol {
    typedef T TT;
    static constexpr bool P_IS_A = false;
    static constexpr bool SHARE_Q = true;
    static constexpr bool HAS_BIAS = false;
    static constexpr bool TAB = false, TAB_CHUNK = false;
    // P: Wc[(g*KK*cg + p) * og + k]
    struct PK { int base; bool ok; };
    __device__ static PK pk(const GemmArgs& a, const Ctx& c, int k)
    {
        return PK{c.grp * a.KK * a.cg * a.og + k, k < c.kend};
    }
    __device__ static T p_sk(const GemmArgs& a, const Buf<T>& B, const Ctx&, const PK& s, int p)
    {
        return B.at(s.ok & (p < a.Pdim), s.base + p * a.og);
    }
    typedef RowOk PV;
    __device__ static PV pv(const GemmArgs& a, const Ctx& c, int p)
    {
        return PV{(c.grp * a.KK * a.cg + p) * a.og, p < a.Pdim};
    }
    template <class BT>
    __device__ static u32x4 p_kv(const GemmArgs&, const BT& B, const Ctx& c, const PV& s, int k)
    {
        return B.at16(s.ok & (k < c.kend), s.off + k);
    }
    // Q: dy[q * OC + g*og + k]
    struct QK { int off; bool ok; };
    __device__ static QK qk(const GemmArgs& a, const Ctx& c, int k)
    {
        return QK{c.grp * a.og + k, k < c.kend};
    }
    __device__ static T q_sk(const GemmArgs& a, const Buf<T>& B, const Ctx&, const QK& s, int q)
    {
        return B.at(s.ok & (q < a.Qdim), q * a.OC + s.off);
    }
    typedef RowOk QV;
    __device__ static QV qv(const GemmArgs& a, const Ctx& c, int q)
    {
        return QV{q * a.OC + c.grp * a.og, q < a.Qdim};
    }
    template <class BT>
    __device__ static u32x4 q_kv(const GemmArgs&, const BT& B, const Ctx& c, const QV& s, int k)
    {
        return B.at16(s.ok & (k < c.kend), s.off + k);
    }
    __device__ static void store4(const GemmArgs& a, const Ctx& c, int p, int q, f32x4 acc, int np)
    {
        const long long idx = ((long long)c.grp * a.Qdim + q) * a.Pdim + p;
        float* o = static_cast<float*>(a.out) + idx;
        if (np == 4 && a.vec_out) *reinterpret_cast<f32x4*>(o) = acc;
        else for (int i = 0; i < np; ++i) o[i] = acc[i];
    }
    static constexpr bool ROW_EPI = true, EPI_RELU = false, EPI_MASK = false;
    __device__ static long long out_index(const GemmArgs& a, const Ctx& c, int p, int q)
    {
        return ((long long)c.grp * a.Qdim + q) * a.Pdim + p;
    }
    __device__ static bool rows8(const GemmArgs& a) { return a.Pdim % 8 == 0; }
    __device__ static bool out_f32(const GemmArgs&) { return true; }
};

// ------------------------------------------------------------------------------------------
// Convolution weight gradient of one shard (eq. 3, the gradient of the shard's mean loss):
// p = output channel in the group, q = (u, v, ci) with ci innermost plus the extra row
// q = K*K*cg of ones (bias gradient), k = position (n, oh, ow) in the shard.  P = dy^T
// (tensor a), Q = patches^T of x (tensor b).  The per-k part of the patch offset comes from the
// table.  blockIdx.z = (shard * splits + split) * G + group.
// ------------------------------------------------------------------------------------------
template <typename T> struct ConvWgrad {
    typedef T TT;
    static constexpr bool P_IS_A = true;
    static constexpr bool SHARE_Q = true;
    static constexpr bool INTERLEAVE = true;
    static constexpr bool HAS_BIAS = false;
    static constexpr bool TAB = true, TAB_CHUNK = false;
    // entry for position k of the shard: the offset of x[b0 + n][oh*S - PD][ow*S - PD][0] and
    // the window origin (oh*S - PD, ow*S - PD)
    __device__ static TabEnt tab_entry(const GemmArgs& a, const Ctx& c, int k)
    {
        if (k >= c.kend) return TabEnt{0, (short)-kFar, (short)-kFar};
        const unsigned b = fdiv(a.fd_ohw, (unsigned)k), hw = (unsigned)k - b * (unsigned)(a.OH * a.OW);
        const unsigned oh = fdiv(a.fd_ow, hw), ow = hw - oh * (unsigned)a.OW;
        const int h0 = (int)oh * a.S - a.PD, w0 = (int)ow * a.S - a.PD;
        return TabEnt{(((c.b0 + (int)b) * a.H + h0) * a.W + w0) * a.C, (short)h0, (short)w0};
    }
    // P: dy[(b0*OH*OW + k) * OC + g*og + p]
    typedef RowOk PR;
    __device__ static PR pr(const GemmArgs& a, const Ctx& c, int p)
    {
        return PR{c.b0 * a.OH * a.OW * a.OC + c.grp * a.og + p, p < a.Pdim};
    }
    __device__ static T p_sr(const GemmArgs& a, const Buf<T>& B, const Ctx& c, const PR& s, int k)
    {
        return B.at(s.ok & (k < c.kend), s.off + k * a.OC);
    }
    typedef RowOk PC;
    __device__ static PC pc(const GemmArgs& a, const Ctx& c, int p0) { return pr(a, c, p0); }
    __device__ static u32x4 p_rv(const GemmArgs& a, const Buf<T>& B, const Ctx& c, const PC& s, int k)
    {
        return B.at16(s.ok & (k < c.kend), s.off + k * a.OC);
    }
    // Q: x at window tap (u, v) of position k, channel g*cg + ci
    struct QR { int off, u, v; bool ok, bias; };
    __device__ static QR qr(const GemmArgs& a, const Ctx& c, int q)
    {
        const int nq = a.KK * a.cg;
        QR s;
        s.ok = q < nq;
        s.bias = q == nq;
        const int qq = s.ok ? q : 0;
        const int kc = a.K * a.cg;
        s.u = qq / kc;
        const int rem = qq - s.u * kc;
        s.v = rem / a.cg;
        const int ci = rem - s.v * a.cg;
        s.off = (s.u * a.W + s.v) * a.C + c.grp * a.cg + ci;
        return s;
    }
    __device__ static T q_sr(const GemmArgs& a, const Buf<T>& B, const Ctx& c, const QR& s, int k)
    {
        const TabEnt e = ld_tab(c.tab + (k - c.kbeg));
        const int hi = e.u + s.u, wi = e.v + s.v;
        const T x = B.at(s.ok & inside(hi, wi, a.H, a.W), e.off + s.off);
        return s.bias ? (k < c.kend ? one<T>() : zero<T>()) : x;
    }
    typedef QR QC;
    __device__ static QC qc(const GemmArgs& a, const Ctx& c, int q0) { return qr(a, c, q0); }
    __device__ static u32x4 q_rv(const GemmArgs& a, const Buf<T>& B, const Ctx& c, const QC& s, int k)
    {
        const TabEnt e = ld_tab(c.tab + (k - c.kbeg));
        const int hi = e.u + s.u, wi = e.v + s.v;
        const u32x4 x = B.at16(s.ok & inside(hi, wi, a.H, a.W), e.off + s.off);
        if (s.bias) return k < c.kend ? one_chunk<T>() : u32x4{0u, 0u, 0u, 0u};
        return x;
    }
    // grads[r][w_off + co * cg*KK + ci*KK + u*K + v] (logical layout) or the bias
    __device__ static void store4(const GemmArgs& a, const Ctx& c, int p, int q, f32x4 acc, int np)
    {
        const int nq = a.KK * a.cg;
        float* g = static_cast<float*>(a.out) + (long long)c.r * a.out_ld;
        const int co = c.grp * a.og + p;
        if (q == nq) {
            for (int i = 0; i < np; ++i) g[a.bias_off + co + i] = acc[i];
            return;
        }
        const int kc = a.K * a.cg;
        const int u = q / kc, rem = q - u * kc, v = rem / a.cg, ci = rem - v * a.cg;
        const long long col = (long long)ci * a.KK + u * a.K + v;
        for (int i = 0; i < np; ++i) g[a.out_off + (long long)(co + i) * nq + col] = acc[i];
    }
};

// ------------------------------------------------------------------------------------------
// First-layer convolution over the padded input X'[n][Hp][Wp][Cp] (groups 1): k = (u, j),
// j < RUN, and the K*Cp inputs of kernel row u of output position q are contiguous at
// X'[n][oh*S + u][ow*S][0..], so every operand load is 16 bytes and needs no bounds test
// (the border of X' holds the zero padding).  Taps j >= K*Cp read neighbouring inputs and meet
// zero weights.
// ------------------------------------------------------------------------------------------
template <typename T> struct ConvFwdRun {
    typedef T TT;
    static constexpr bool P_IS_A = false;
    static constexpr bool SHARE_Q = true;
    static constexpr bool TAB = true, TAB_CHUNK = true;
    // entry for the chunk starting at k: offset of (u, j) from the window origin
    __device__ static TabEnt tab_entry(const GemmArgs& a, const Ctx& c, int k)
    {
        if (k >= c.kend) return TabEnt{0, 0, 0};
        const int u = (int)fdiv(a.fd_run, (unsigned)k), j = k - u * a.RUN;
        return TabEnt{u * a.Wp * a.Cp + j, 0, 0};
    }
    // P: Wr[p * Kdim + k]
    typedef RowOk PV;
    __device__ static PV pv(const GemmArgs& a, const Ctx&, int p) { return PV{p * a.Kdim, p < a.Pdim}; }
    template <class BT>
    __device__ static u32x4 p_kv(const GemmArgs&, const BT& B, const Ctx& c, const PV& s, int k)
    {
        return B.at16(s.ok & (k < c.kend), s.off + k);
    }
    // Q: window origin of output position q
    typedef RowOk QV;
    __device__ static QV qv(const GemmArgs& a, const Ctx&, int q)
    {
        const bool ok = q < a.Qdim;
        const unsigned qq = ok ? q : 0;
        const unsigned b = fdiv(a.fd_ohw, qq), hw = qq - b * (unsigned)(a.OH * a.OW);
        const unsigned oh = fdiv(a.fd_ow, hw), ow = hw - oh * (unsigned)a.OW;
        return QV{(((int)b * a.Hp + (int)oh * a.S) * a.Wp + (int)ow * a.S) * a.Cp, ok};
    }
    template <class BT>
    __device__ static u32x4 q_kv(const GemmArgs&, const BT& B, const Ctx& c, const QV& s, int k)
    {
        const TabEnt e = ld_tab(c.tab + (k - c.kbeg) / (16 / (int)sizeof(T)));
        return B.at16(s.ok, s.off + e.off);
    }
    static constexpr bool HAS_BIAS = true;
    __device__ static int bias_index(const GemmArgs&, const Ctx&, int p) { return p; }
    __device__ static void store4(const GemmArgs& a, const Ctx& c, int p, int q, f32x4 acc, int np)
    {
        ConvFwd<T>::store4(a, c, p, q, acc, np);
    }
    static constexpr bool ROW_EPI = true, EPI_RELU = true, EPI_MASK = false;
    __device__ static long long out_index(const GemmArgs& a, const Ctx& c, int p, int q)
    {
        return ConvFwd<T>::out_index(a, c, p, q);
    }
    __device__ static bool rows8(const GemmArgs& a) { return ConvFwd<T>::rows8(a); }
    __device__ static bool out_f32(const GemmArgs& a) { return a.out_f32; }
};

// Weight gradient of one shard for the same layer: p = output channel, q = (u, j) plus the
// bias row q = K*RUN, k = position in the shard.  Outputs for padding taps are discarded.
template <typename T> struct ConvWgradRun {
    typedef T TT;
    static constexpr bool P_IS_A = true;
    static constexpr bool SHARE_Q = true;
    static constexpr bool HAS_BIAS = false;
    static constexpr bool TAB = true, TAB_CHUNK = false;
    // entry for position k of the shard: offset of its window origin in X'
    __device__ static TabEnt tab_entry(const GemmArgs& a, const Ctx& c, int k)
    {
        if (k >= c.kend) return TabEnt{0, 0, 0};
        const unsigned b = fdiv(a.fd_ohw, (unsigned)k), hw = (unsigned)k - b * (unsigned)(a.OH * a.OW);
        const unsigned oh = fdiv(a.fd_ow, hw), ow = hw - oh * (unsigned)a.OW;
        return TabEnt{(((c.b0 + (int)b) * a.Hp + (int)oh * a.S) * a.Wp + (int)ow * a.S) * a.Cp, 0, 0};
    }
    // P: dy^T, as for ConvWgrad
    typedef RowOk PR;
    __device__ static PR pr(const GemmArgs& a, const Ctx& c, int p)
    {
        return PR{c.b0 * a.OH * a.OW * a.OC + p, p < a.Pdim};
    }
    __device__ static T p_sr(const GemmArgs& a, const Buf<T>& B, const Ctx& c, const PR& s, int k)
    {
        return B.at(s.ok & (k < c.kend), s.off + k * a.OC);
    }
    typedef RowOk PC;
    __device__ static PC pc(const GemmArgs& a, const Ctx& c, int p0) { return pr(a, c, p0); }
    __device__ static u32x4 p_rv(const GemmArgs& a, const Buf<T>& B, const Ctx& c, const PC& s, int k)
    {
        return B.at16(s.ok & (k < c.kend), s.off + k * a.OC);
    }
    // Q: X' at (u, j) of the window of position k
    struct QR { int off; bool ok, bias; };
    __device__ static QR qr(const GemmArgs& a, const Ctx&, int q)
    {
        const int nq = a.K * a.RUN;
        const int qq = q < nq ? q : 0;
        const int u = (int)fdiv(a.fd_run, (unsigned)qq), j = qq - u * a.RUN;
        return QR{u * a.Wp * a.Cp + j, q < nq, q == nq};
    }
    __device__ static T q_sr(const GemmArgs& a, const Buf<T>& B, const Ctx& c, const QR& s, int k)
    {
        const TabEnt e = ld_tab(c.tab + (k - c.kbeg));
        const T x = B.at(s.ok, e.off + s.off);
        return s.bias ? (k < c.kend ? one<T>() : zero<T>()) : x;
    }
    typedef QR QC;
    __device__ static QC qc(const GemmArgs& a, const Ctx& c, int q0) { return qr(a, c, q0); }
    __device__ static u32x4 q_rv(const GemmArgs& a, const Buf<T>& B, const Ctx& c, const QC& s, int k)
    {
        const TabEnt e = ld_tab(c.tab + (k - c.kbeg));
        const u32x4 x = B.at16(s.ok, e.off + s.off);
        if (s.bias) return k < c.kend ? one_chunk<T>() : u32x4{0u, 0u, 0u, 0u};
        return x;
    }
    // grads[r][w_off + co * C*K*K + ci*K*K + u*K + v] for the real taps, or the bias
    __device__ static void store4(const GemmArgs& a, const Ctx& c, int p, int q, f32x4 acc, int np)
    {
        const int nq = a.K * a.RUN;
        float* g = static_cast<float*>(a.out) + (long long)c.r * a.out_ld;
        if (q == nq) {
            for (int i = 0; i < np; ++i) g[a.bias_off + p + i] = acc[i];
            return;
        }
        const int u = q / a.RUN, j = q - u * a.RUN, v = j / a.Cp, ci = j - v * a.Cp;
        if (v >= a.K || ci >= a.C) return;
        const int nw = a.C * a.KK;
        const long long col = (long long)ci * a.KK + u * a.K + v;
        for (int i = 0; i < np; ++i) g[a.out_off + (long long)(p + i) * nw + col] = acc[i];
    }
};

// ------------------------------------------------------------------------------------------
// Fully connected layers: y = W x + b.  Inputs after a spatial layer are in (h, w, c) order and
// the prepared weights follow that order.
// ------------------------------------------------------------------------------------------

// Forward: p = output unit o, q = sample, k = input feature.  P = W (tensor b), Q = x (tensor a).
template <typename T> struct FcFwd {
    typedef T TT;
    static constexpr bool P_IS_A = false;
    static constexpr bool SHARE_Q = false;
    static constexpr bool TAB = false, TAB_CHUNK = false;
    static constexpr bool DEEP_PREFETCH = sizeof(T) == 2;  // few blocks: loads 3 k tiles ahead
    struct PK { int k; bool ok; };
    __device__ static PK pk(const GemmArgs&, const Ctx& c, int k) { return PK{k, k < c.kend}; }
    __device__ static T p_sk(const GemmArgs& a, const Buf<T>& B, const Ctx&, const PK& s, int p)
    {
        return B.at(s.ok & (p < a.Pdim), p * a.Kdim + s.k);
    }
    typedef RowOk PV;
    __device__ static PV pv(const GemmArgs& a, const Ctx&, int p) { return PV{p * a.Kdim, p < a.Pdim}; }
    template <class BT>
    __device__ static u32x4 p_kv(const GemmArgs&, const BT& B, const Ctx& c, const PV& s, int k)
    {
        return B.at16(s.ok & (k < c.kend), s.off + k);
    }
    typedef PK QK;
    __device__ static QK qk(const GemmArgs&, const Ctx& c, int k) { return QK{k, k < c.kend}; }
    __device__ static T q_sk(const GemmArgs& a, const Buf<T>& B, const Ctx&, const QK& s, int q)
    {
        return B.at(s.ok & (q < a.Qdim), q * a.Kdim + s.k);
    }
    typedef RowOk QV;
    __device__ static QV qv(const GemmArgs& a, const Ctx&, int q) { return QV{q * a.Kdim, q < a.Qdim}; }
    template <class BT>
    __device__ static u32x4 q_kv(const GemmArgs&, const BT& B, const Ctx& c, const QV& s, int k)
    {
        return B.at16(s.ok & (k < c.kend), s.off + k);
    }
    static constexpr bool HAS_BIAS = true;
    __device__ static int bias_index(const GemmArgs&, const Ctx&, int p) { return p; }
    // y[q][p] = acc (bias included), ReLU
    __device__ static void store4(const GemmArgs& a, const Ctx&, int p, int q, f32x4 acc, int np)
    {
        float v[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = a.relu ? fmaxf(acc[i], 0.f) : acc[i];
        store_vals<T>(a.out, a.out_f32, q * a.Pdim + p, v, np, a.vec_out);
    }
    // staged row epilogue (see igemm_kernel): rows q contiguous along p
    static constexpr bool ROW_EPI = true, EPI_RELU = true, EPI_MASK = false;
    __device__ static long long out_index(const GemmArgs& a, const Ctx&, int p, int q)
    {
        return (long long)q * a.Pdim + p;
    }
    __device__ static bool rows8(const GemmArgs& a) { return a.Pdim % 8 == 0; }
    __device__ static bool out_f32(const GemmArgs& a) { return a.out_f32; }
};

// Data gradient: p = input feature i, q = sample, k = output unit o.  P = W^T (tensor b, rows
// i contiguous in W[o][i]), Q = dy (tensor a).
template <typename T> struct FcDgrad {
    typedef T TT;
    static constexpr bool P_IS_A = false;
    static constexpr bool SHARE_Q = false;
    static constexpr bool HAS_BIAS = false;
    static constexpr bool TAB = false, TAB_CHUNK = false;
    typedef RowOk PR;
    __device__ static PR pr(const GemmArgs& a, const Ctx&, int p) { return PR{p, p < a.Pdim}; }
    __device__ static T p_sr(const GemmArgs& a, const Buf<T>& B, const Ctx& c, const PR& s, int k)
    {
        return B.at(s.ok & (k < c.kend), k * a.Pdim + s.off);
    }
    typedef RowOk PC;
    __device__ static PC pc(const GemmArgs& a, const Ctx&, int p0) { return PC{p0, p0 < a.Pdim}; }
    __device__ static u32x4 p_rv(const GemmArgs& a, const Buf<T>& B, const Ctx& c, const PC& s, int k)
    {
        return B.at16(s.ok & (k < c.kend), k * a.Pdim + s.off);
    }
    struct QK { int k; bool ok; };
    __device__ static QK qk(const GemmArgs&, const Ctx& c, int k) { return QK{k, k < c.kend}; }
    __device__ static T q_sk(const GemmArgs& a, const Buf<T>& B, const Ctx&, const QK& s, int q)
    {
        return B.at(s.ok & (q < a.Qdim), q * a.Kdim + s.k);
    }
    typedef RowOk QV;
    __device__ static QV qv(const GemmArgs& a, const Ctx&, int q) { return QV{q * a.Kdim, q < a.Qdim}; }
    template <class BT>
    __device__ static u32x4 q_kv(const GemmArgs&, const BT& B, const Ctx& c, const QV& s, int k)
    {
        return B.at16(s.ok & (k < c.kend), s.off + k);
    }
    // dx[q][p] = acc, times the ReLU mask of the layer below
    __device__ static void store4(const GemmArgs& a, const Ctx&, int p, int q, f32x4 acc, int np)
    {
        const int idx = q * a.Pdim + p;
        float v[4] = {acc[0], acc[1], acc[2], acc[3]};
        apply_mask<T>(a, idx, v, np);
        store_vals<T>(a.out, false, idx, v, np, a.vec_out);
    }
    static constexpr bool ROW_EPI = true, EPI_RELU = false, EPI_MASK = true;
    __device__ static long long out_index(const GemmArgs& a, const Ctx&, int p, int q)
    {
        return (long long)q * a.Pdim + p;
    }
    __device__ static bool rows8(const GemmArgs& a) { return a.Pdim % 8 == 0; }
    __device__ static bool out_f32(const GemmArgs&) { return false; }
};

// Weight gradient of one shard: p = input feature i (logical (c, h, w) order) plus the bias
// row p = IN, q = output unit o, k = sample in the shard.  P = x^T (tensor b), Q = dy^T
// (tensor a); both row-contiguous.  When the input is stored in (h, w, c) order (perm_c,
// perm_hw > 1) the row-fast scalar loader maps each logical row to its stored column, so the
// gradient is written in logical order either way.  blockIdx.z as for convolutions (G = 1).
template <typename T> struct FcWgrad {
    typedef T TT;
    static constexpr bool P_IS_A = false;
    // neighbouring blocks of an XCD take the p tiles of one q tile: they write consecutive
    // 512-byte pieces of the same gradient rows (the operands, K = one shard's samples, are
    // small); AlexNet FC6 with the fused update 0.429 -> 0.400 ms
    static constexpr bool SHARE_Q = true;
    static constexpr bool HAS_BIAS = false;
    static constexpr bool TAB = false, TAB_CHUNK = false;
    struct PR { int i; bool ok, bias; };
    __device__ static PR pr(const GemmArgs& a, const Ctx&, int p)
    {
        int i = p;
        if (a.perm_c > 1 && a.perm_hw > 1 && p < a.C) {
            const int ch = p / a.perm_hw, hw = p - ch * a.perm_hw;
            i = hw * a.perm_c + ch;
        }
        return PR{i, p < a.C, p == a.C};
    }
    __device__ static T p_sr(const GemmArgs& a, const Buf<T>& B, const Ctx& c, const PR& s, int k)
    {
        const bool kok = k < c.kend;
        const T x = B.at(s.ok & kok, (c.b0 + k) * a.C + s.i);
        return s.bias ? (kok ? one<T>() : zero<T>()) : x;
    }
    // (16-byte loads only for inputs in logical order)
    typedef PR PC;
    __device__ static PC pc(const GemmArgs& a, const Ctx&, int p0) { return PC{p0, p0 < a.C, p0 == a.C}; }
    __device__ static u32x4 p_rv(const GemmArgs& a, const Buf<T>& B, const Ctx& c, const PC& s, int k)
    {
        const bool kok = k < c.kend;
        const u32x4 x = B.at16(s.ok & kok, (c.b0 + k) * a.C + s.i);
        if (s.bias) return kok ? one_chunk<T>() : u32x4{0u, 0u, 0u, 0u};
        return x;
    }
    typedef RowOk QR;
    __device__ static QR qr(const GemmArgs& a, const Ctx&, int q) { return QR{q, q < a.Qdim}; }
    __device__ static T q_sr(const GemmArgs& a, const Buf<T>& B, const Ctx& c, const QR& s, int k)
    {
        return B.at(s.ok & (k < c.kend), (c.b0 + k) * a.Qdim + s.off);
    }
    typedef RowOk QC;
    __device__ static QC qc(const GemmArgs& a, const Ctx& c, int q0) { return qr(a, c, q0); }
    __device__ static u32x4 q_rv(const GemmArgs& a, const Buf<T>& B, const Ctx& c, const QC& s, int k)
    {
        return B.at16(s.ok & (k < c.kend), (c.b0 + k) * a.Qdim + s.off);
    }
    // grads[r][w_off + o * IN + i], or the bias
    static constexpr bool ROW_STORE = true;  // row o is contiguous along i (staged row store)
    __device__ static int row_len(const GemmArgs& a) { return a.C; }
    __device__ static float* row_out(const GemmArgs& a, const Ctx& c, int q)
    {
        return static_cast<float*>(a.out) + (long long)c.r * a.out_ld + a.out_off +
               (long long)q * a.C;
    }
    __device__ static void store4(const GemmArgs& a, const Ctx& c, int p, int q, f32x4 acc, int np)
    {
        float* g = static_cast<float*>(a.out) + (long long)c.r * a.out_ld;
        const long long row = a.out_off + (long long)q * a.C;
        if (p + 3 < a.C && a.vec_out) {
            *reinterpret_cast<f32x4*>(g + row + p) = acc;
            return;
        }
        for (int i = 0; i < np; ++i) {
            if (p + i == a.C) g[a.bias_off + q] = acc[i];
            else g[row + p + i] = acc[i];
        }
    }
    // parameter of output (p, q) in a gradient row (W[q][p], or b[q] for the bias row), -1 outside
    __device__ static long long param_index(const GemmArgs& a, int p, int q)
    {
        if (p < a.C) return a.out_off + (long long)q * a.C + p;
        return p == a.C ? a.bias_off + q : -1;
    }
};

// The same weight gradient for all R shards of one output tile per block, followed by the
// average of the R stored values and the optimizer step of the tile's parameters (Sec. III-D.2:
// each layer's reduction and update; the momentum rule of the stand-alone kernel, element by
// element the same arithmetic).
template <typename T> struct FcWgradUpd : FcWgrad<T> {
    static constexpr bool FUSE_UPDATE = true;
};

}  // namespace mtx
