// Internal declarations shared by the host orchestration (api.hip) and the kernel files.
#pragma once

#include <hip/hip_runtime.h>
#include <cstddef>
#include <cstdint>

namespace mtx {

enum Dt { DT_F32 = 0, DT_BF16 = 1 };

// Geometry of one convolution (or of a fully connected layer viewed as C=in, H=W=K=1).
struct ConvGeom {
    int N;            // images in the launch (whole batch for fwd/dgrad, one shard for wgrad)
    int C, H, W;      // input
    int OC, OH, OW;   // output
    int K, S, PD, G;  // kernel, stride, padding, groups
};

// Implicit-GEMM arguments.  Each operation (see igemm.hip) reads the fields it needs.
struct GemmArgs {
    const void* a;         // activation-like operand (x, dy or X)
    const void* b;         // weights or second activation operand
    void* out;             // output (activation, data gradient, or fp32 gradient rows)
    const float* bias;     // forward: fp32 bias [OC]
    const void* mask;      // data gradient: the previous layer's stored output (ReLU mask)
    float* partial;        // weight gradient with split K: fp32 partial sums
    long long out_ld;      // weight gradient: elements between shard gradient rows
    long long out_off;     // weight gradient: offset of this layer's W in a gradient row
    long long bias_off;    // weight gradient: offset of this layer's b in a gradient row
    int N, C, H, W, OC, OH, OW, K, S, PD, G;
    int cg, og, KK;        // C/G, OC/G, K*K
    int Pdim, Qdim, Kdim;  // GEMM sizes: output rows, output columns, reduction length
    int splits;            // reduction splits (blockIdx.z = (shard * splits + split) * G + group)
    int kchunk;            // reduction length of one split (multiple of the k tile)
    int R;                 // weight gradient: shards in the launch
    int relu;              // forward: apply ReLU
    int out_f32;           // forward: output stored as fp32 (otherwise the compute type)
    int mask_f32;          // data gradient: mask tensor is fp32 (otherwise the compute type)
    unsigned a_bytes;      // size of tensor a in bytes (buffer-load range)
    unsigned b_bytes;      // size of tensor b in bytes
};

// GEMM view of one operation: P output rows, Q output columns, K reduction length, Z blocks
// along blockIdx.z before reduction splits (groups x shards).
struct GemmDims {
    int P, Q, K, Z;
    bool allow_split;
};
// Launch shape: 32*FP x 32*FQ output tile, BK reduction tile, reduction splits of kchunk.
struct GemmPlan {
    int FP, FQ, BK, splits, kchunk;
};
GemmPlan plan_gemm(int dt, int Pdim, int Qdim, int Kdim, int zdim, bool allow_split);
GemmPlan plan_for(int dt, const GemmDims& d);
size_t partial_elems(int dt, const GemmDims& d);  // fp32 partial sums a launch needs (0 if none)
GemmDims conv_fwd_dims(const ConvGeom& g);
GemmDims conv_dgrad_dims(const ConvGeom& g);
GemmDims conv_wgrad_dims(const ConvGeom& g, int R);
GemmDims conv_dgrad_col_dims(const ConvGeom& g);
size_t conv_dgrad_col_elems(const ConvGeom& g);
bool conv_dgrad_use_col(const ConvGeom& g);  // data gradient through col + col2im
GemmDims fc_fwd_dims(int B, int IN, int OUT);
GemmDims fc_dgrad_dims(int B, int IN, int OUT);
GemmDims fc_wgrad_dims(int Nb, int R, int IN, int OUT);

// `partial` is fp32 scratch of at least partial_elems() elements (may be null when 0).
hipError_t conv_fwd(Dt dt, const ConvGeom& g, const void* x, const void* w, const float* bias,
                    void* y, bool y_f32, bool relu, float* partial, hipStream_t s);
hipError_t conv_dgrad(Dt dt, const ConvGeom& g, const void* dy, const void* w, void* dx,
                      const void* mask, bool mask_f32, float* partial, hipStream_t s);
// Data gradient through an fp32 col buffer of conv_dgrad_col_elems() elements.
hipError_t conv_dgrad_col(Dt dt, const ConvGeom& g, const void* dy, const void* w, void* dx,
                          const void* mask, bool mask_f32, float* col, float* partial,
                          hipStream_t s);
// Weight and bias gradient of R shards of g.N images each; x and dy point at the first shard.
hipError_t conv_wgrad(Dt dt, const ConvGeom& g, int R, const void* x, const void* dy,
                      float* grads, long long ld, long long w_off, long long b_off,
                      float* partial, hipStream_t s);
hipError_t fc_fwd(Dt dt, int B, int IN, int OUT, const void* x, const void* w, const float* bias,
                  void* y, bool y_f32, bool relu, float* partial, hipStream_t s);
hipError_t fc_dgrad(Dt dt, int B, int IN, int OUT, const void* dy, const void* w, void* dx,
                    const void* mask, bool mask_f32, float* partial, hipStream_t s);
hipError_t fc_wgrad(Dt dt, int Nb, int R, int IN, int OUT, const void* x, const void* dy,
                    float* grads, long long ld, long long w_off, long long b_off, float* partial,
                    hipStream_t s);

// elementwise.hip
hipError_t cast_bf16(const float* src, void* dst, size_t n, hipStream_t s);
hipError_t pool_fwd(Dt dt, int N, int C, int H, int W, int K, int S, const void* x, void* y,
                    uint8_t* argmax, hipStream_t s);
hipError_t pool_bwd(Dt dt, int N, int C, int H, int W, int K, int S, const uint8_t* argmax,
                    const void* dy, void* dx, const void* mask, bool mask_f32, hipStream_t s);
// Softmax cross-entropy of B rows; with loss_out set, also the batch-mean loss (block_sums holds
// ceil(B/4) floats; *sync must be 0 before the first launch and is 0 again after every launch).
hipError_t softmax_xent(Dt dt, int B, int NC, int Nb, const float* logits,
                        const int32_t* labels, void* dz, float* block_sums, unsigned* sync,
                        float* loss_out, hipStream_t s);
hipError_t average_update(const float* grads, int R, size_t n, size_t ld, float* w, float* v,
                          float lr, float mu, float* avg, bool update, hipStream_t s);

}  // namespace mtx
