// Weight-gradient launches (per shard, bias gradient included): convolution and fully
// connected.
#include "igemm_ops.h"

namespace mtx {

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
    const GemmDims d = conv_wgrad_dims(dt, g, R);
    a.Pdim = d.P; a.Qdim = d.Q; a.Kdim = d.K;
    const GemmPlan p = plan_for(dt, d);
    const bool pv = a.og % vec_elems(dt) == 0, qv = a.cg % vec_elems(dt) == 0;
    if (dt == DT_F32) {
        typedef ConvWgrad<float> Op;
        if (pv && qv) return run_gemm<Op, L_RT, L_RT>(a, p, d.Z, partial, s);
        if (pv) return run_gemm<Op, L_RT, L_SR>(a, p, d.Z, partial, s);
        if (qv) return run_gemm<Op, L_SR, L_RT>(a, p, d.Z, partial, s);
        return run_gemm<Op, L_SR, L_SR>(a, p, d.Z, partial, s);
    }
    typedef ConvWgrad<bf16_t> Op;
    if (pv && qv) return run_gemm<Op, L_RT, L_RT>(a, p, d.Z, partial, s);
    if (pv) return run_gemm<Op, L_RT, L_SR>(a, p, d.Z, partial, s);
    if (qv) return run_gemm<Op, L_SR, L_RT>(a, p, d.Z, partial, s);
    return run_gemm<Op, L_SR, L_SR>(a, p, d.Z, partial, s);
}

hipError_t conv_wgrad_run(Dt dt, const ConvGeom& g, const RunGeom& r, int R, const void* xp,
                          const void* dy, float* grads, long long ld, long long w_off,
                          long long b_off, float* partial, hipStream_t s)
{
    if (g.G != 1) return hipErrorInvalidValue;
    GemmArgs a = conv_args(g);
    a.Hp = r.Hp; a.Wp = r.Wp; a.Cp = r.Cp; a.RUN = r.RUN;
    a.fd_run = make_fastdiv((unsigned)r.RUN);
    a.a = dy; a.b = xp; a.out = grads; a.out_ld = ld; a.out_off = w_off; a.bias_off = b_off;
    a.R = R;
    const unsigned es = dt == DT_F32 ? 4 : 2;
    a.a_bytes = (unsigned)((size_t)R * g.N * g.OC * g.OH * g.OW * es);
    a.b_bytes = (unsigned)((size_t)R * g.N * r.Hp * r.Wp * r.Cp * es);
    const GemmDims d = conv_wgrad_run_dims(dt, g, r, R);
    a.Pdim = d.P; a.Qdim = d.Q; a.Kdim = d.K;
    const GemmPlan p = plan_for(dt, d);
    const bool pv = g.OC % vec_elems(dt) == 0;
    if (dt == DT_F32) {
        typedef ConvWgradRun<float> Op;
        if (pv) return run_gemm<Op, L_RT, L_RT>(a, p, d.Z, partial, s);
        return run_gemm<Op, L_SR, L_RT>(a, p, d.Z, partial, s);
    }
    typedef ConvWgradRun<bf16_t> Op;
    if (pv) return run_gemm<Op, L_RT, L_RT>(a, p, d.Z, partial, s);
    return run_gemm<Op, L_SR, L_RT>(a, p, d.Z, partial, s);
}

hipError_t fc_wgrad(Dt dt, int Nb, int R, int IN, int OUT, int perm_c, int perm_hw,
                    const void* x, const void* dy, float* grads, long long ld, long long w_off,
                    long long b_off, float* partial, hipStream_t s)
{
    GemmArgs a{};
    a.a = dy; a.b = x; a.out = grads; a.out_ld = ld; a.out_off = w_off; a.bias_off = b_off;
    a.N = Nb; a.C = IN; a.OC = OUT; a.G = 1; a.R = R; a.perm_c = perm_c; a.perm_hw = perm_hw;
    a.vec_out = IN % 4 == 0 && w_off % 4 == 0 && ld % 4 == 0;
    const unsigned es = dt == DT_F32 ? 4 : 2;
    a.a_bytes = (unsigned)((size_t)R * Nb * OUT * es);
    a.b_bytes = (unsigned)((size_t)R * Nb * IN * es);
    const GemmDims d = fc_wgrad_dims(dt, Nb, R, IN, OUT);
    a.Pdim = d.P; a.Qdim = d.Q; a.Kdim = d.K;
    const GemmPlan p = plan_for(dt, d);
    const bool perm = perm_c > 1 && perm_hw > 1;
    const bool pv = IN % vec_elems(dt) == 0 && !perm, qv = OUT % vec_elems(dt) == 0;
    if (dt == DT_F32) {
        typedef FcWgrad<float> Op;
        if (pv && qv) return run_gemm<Op, L_RT, L_RT>(a, p, d.Z, partial, s);
        if (pv) return run_gemm<Op, L_RT, L_SR>(a, p, d.Z, partial, s);
        if (qv) return run_gemm<Op, L_SR, L_RT>(a, p, d.Z, partial, s);
        return run_gemm<Op, L_SR, L_SR>(a, p, d.Z, partial, s);
    }
    typedef FcWgrad<bf16_t> Op;
    if (pv && qv) return run_gemm<Op, L_RT, L_RT>(a, p, d.Z, partial, s);
    if (pv) return run_gemm<Op, L_RT, L_SR>(a, p, d.Z, partial, s);
    if (qv) return run_gemm<Op, L_SR, L_RT>(a, p, d.Z, partial, s);
    return run_gemm<Op, L_SR, L_SR>(a, p, d.Z, partial, s);
}

// The fused form (one block per output tile for all R shards, then the average + update of the
// tile's parameters) is planned with one block row per tile (Z = 1) and needs an unsplit
// reduction; then it replaces fc_wgrad and this layer's share of the average + update.
static GemmDims fc_wgrad_update_dims(int dt, int Nb, int R, int IN, int OUT)
{
    GemmDims d = fc_wgrad_dims(dt, Nb, R, IN, OUT);
    d.Z = 1;
    return d;
}

bool fc_wgrad_update_ok(Dt dt, int Nb, int R, int IN, int OUT)
{
    // Only for layers large enough to be bound by their gradient rows (at least 2^20 parameters),
    // planned with 128 x 128 tiles (the staged row store) and enough of them to keep two blocks
    // per compute unit busy with one block per tile.  Measured: LeNet's 400 K-parameter fc layer
    // fused took the step from 0.154 to 0.174 ms; AlexNet's FC8 (4 M parameters, 64 x 128 tiles)
    // 0.105 ms fused against 0.065 ms for its weight gradient and share of the average; FC6 and
    // FC7 fused took the step from 3.21 to 3.10 ms.
    const GemmDims d = fc_wgrad_update_dims(dt, Nb, R, IN, OUT);
    const GemmPlan g = plan_for(dt, d);
    const long long tiles = (long long)((d.P + 32 * g.FP - 1) / (32 * g.FP)) *
                            ((d.Q + 32 * g.FQ - 1) / (32 * g.FQ));
    return g.splits == 1 && g.FP == 4 && g.FQ == 4 && R >= 1 && tiles >= 512 &&
           (long long)(IN + 1) * OUT >= (1ll << 20);
}

hipError_t fc_wgrad_update(Dt dt, int Nb, int R, int IN, int OUT, int perm_c, int perm_hw,
                           const void* x, const void* dy, float* grads, long long ld,
                           long long w_off, long long b_off, float* w, float* v, float* avg,
                           float lr, float mu, hipStream_t s)
{
    if (!fc_wgrad_update_ok(dt, Nb, R, IN, OUT)) return hipErrorInvalidValue;
    GemmArgs a{};
    a.a = dy; a.b = x; a.out = grads; a.out_ld = ld; a.out_off = w_off; a.bias_off = b_off;
    a.N = Nb; a.C = IN; a.OC = OUT; a.G = 1; a.R = R; a.perm_c = perm_c; a.perm_hw = perm_hw;
    a.vec_out = IN % 4 == 0 && w_off % 4 == 0 && ld % 4 == 0;
    a.upd_w = w; a.upd_v = mu != 0.0f ? v : nullptr; a.upd_avg = avg;
    a.upd_lr = lr; a.upd_mu = mu;
    const unsigned es = dt == DT_F32 ? 4 : 2;
    a.a_bytes = (unsigned)((size_t)R * Nb * OUT * es);
    a.b_bytes = (unsigned)((size_t)R * Nb * IN * es);
    const GemmDims d = fc_wgrad_update_dims(dt, Nb, R, IN, OUT);
    a.Pdim = d.P; a.Qdim = d.Q; a.Kdim = d.K;
    const GemmPlan p = plan_for(dt, d);
    const bool perm = perm_c > 1 && perm_hw > 1;
    const bool pv = IN % vec_elems(dt) == 0 && !perm, qv = OUT % vec_elems(dt) == 0;
    if (dt == DT_F32) {
        typedef FcWgradUpd<float> Op;
        if (pv && qv) return run_gemm<Op, L_RT, L_RT>(a, p, 1, nullptr, s);
        if (pv) return run_gemm<Op, L_RT, L_SR>(a, p, 1, nullptr, s);
        if (qv) return run_gemm<Op, L_SR, L_RT>(a, p, 1, nullptr, s);
        return run_gemm<Op, L_SR, L_SR>(a, p, 1, nullptr, s);
    }
    typedef FcWgradUpd<bf16_t> Op;
    if (pv && qv) return run_gemm<Op, L_RT, L_RT>(a, p, 1, nullptr, s);
    if (pv) return run_gemm<Op, L_RT, L_SR>(a, p, 1, nullptr, s);
    if (qv) return run_gemm<Op, L_SR, L_RT>(a, p, 1, nullptr, s);
    return run_gemm<Op, L_SR, L_SR>(a, p, 1, nullptr, s);
}

}  // namespace mtx
