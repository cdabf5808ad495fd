// Forward launches: convolution (implicit GEMM over NHWC activations) and fully connected.
#include "igemm_ops.h"

namespace mtx {

hipError_t conv_fwd(Dt dt, const ConvGeom& g, const void* x, const void* wf, const float* bias,
                    void* y, bool y_f32, bool relu, float* partial, hipStream_t s)
{
    GemmArgs a = conv_args(g);
    a.a = x; a.b = wf; a.out = y; a.bias = bias; a.relu = relu; a.out_f32 = y_f32 || dt == DT_F32;
    a.vec_out = g.OC % 4 == 0 && a.og % 4 == 0;
    const unsigned es = dt == DT_F32 ? 4 : 2;
    a.a_bytes = (unsigned)((size_t)g.N * g.C * g.H * g.W * es);
    a.b_bytes = (unsigned)((size_t)g.OC * a.cg * a.KK * es);
    const GemmDims d = conv_fwd_dims(dt, g);
    a.Pdim = d.P; a.Qdim = d.Q; a.Kdim = d.K;
    const GemmPlan p = plan_for(dt, d);
    const bool v = a.cg % vec_elems(dt) == 0;  // then C (= G*cg) and Kdim are multiples too
    if (dt == DT_F32) {
        if (v) return run_gemm<ConvFwd<float>, L_KD, L_KD>(a, p, d.Z, partial, s);
        return run_gemm<ConvFwd<float>, L_SK, L_SR>(a, p, d.Z, partial, s);
    }
    if (v) return run_gemm<ConvFwd<bf16_t>, L_KV, L_KV>(a, p, d.Z, partial, s);
    return run_gemm<ConvFwd<bf16_t>, L_SK, L_SR>(a, p, d.Z, partial, s);
}

hipError_t conv_fwd_run(Dt dt, const ConvGeom& g, const RunGeom& r, const void* xp,
                        const void* wr, const float* bias, void* y, bool y_f32, bool relu,
                        float* partial, hipStream_t s)
{
    if (g.G != 1) return hipErrorInvalidValue;
    GemmArgs a = conv_args(g);
    a.Hp = r.Hp; a.Wp = r.Wp; a.Cp = r.Cp; a.RUN = r.RUN;
    a.fd_run = make_fastdiv((unsigned)r.RUN);
    a.a = xp; a.b = wr; a.out = y; a.bias = bias; a.relu = relu; a.out_f32 = y_f32 || dt == DT_F32;
    a.vec_out = g.OC % 4 == 0;
    const unsigned es = dt == DT_F32 ? 4 : 2;
    a.a_bytes = (unsigned)((size_t)g.N * r.Hp * r.Wp * r.Cp * es);
    a.b_bytes = (unsigned)((size_t)g.OC * g.K * r.RUN * es);
    const GemmDims d = conv_fwd_run_dims(dt, g, r);
    a.Pdim = d.P; a.Qdim = d.Q; a.Kdim = d.K;
    const GemmPlan p = plan_for(dt, d);
    if (dt == DT_F32) return run_gemm<ConvFwdRun<float>, L_KD, L_KD>(a, p, d.Z, partial, s);
    return run_gemm<ConvFwdRun<bf16_t>, L_KV, L_KV>(a, p, d.Z, partial, s);
}

hipError_t fc_fwd(Dt dt, int B, int IN, int OUT, const void* x, const void* w, const float* bias,
                  void* y, bool y_f32, bool relu, float* partial, hipStream_t s)
{
    GemmArgs a{};
    a.a = x; a.b = w; a.out = y; a.bias = bias; a.relu = relu; a.out_f32 = y_f32 || dt == DT_F32;
    a.N = B; a.C = IN; a.OC = OUT; a.G = 1; a.R = 1; a.perm_c = 1; a.perm_hw = 1;
    a.vec_out = OUT % 4 == 0;
    const unsigned es = dt == DT_F32 ? 4 : 2;
    a.a_bytes = (unsigned)((size_t)B * IN * es);
    a.b_bytes = (unsigned)((size_t)OUT * IN * es);
    const GemmDims d = fc_fwd_dims(dt, B, IN, OUT);
    a.Pdim = d.P; a.Qdim = d.Q; a.Kdim = d.K;
    const GemmPlan p = plan_for(dt, d);
    const bool v = IN % vec_elems(dt) == 0;
    if (dt == DT_F32) {
        if (v) return run_gemm<FcFwd<float>, L_KD, L_KD>(a, p, d.Z, partial, s);
        return run_gemm<FcFwd<float>, L_SK, L_SK>(a, p, d.Z, partial, s);
    }
    if (v) return run_gemm<FcFwd<bf16_t>, L_KV, L_KV>(a, p, d.Z, partial, s);
    return run_gemm<FcFwd<bf16_t>, L_SK, L_SK>(a, p, d.Z, partial, s);
}

}  // namespace mtx
