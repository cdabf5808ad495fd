// Internal declarations shared by the host orchestration (api.hip) and the kernel files.
//
// Data layouts on the device (per step):
//   activations and data gradients of convolution and pooling layers: NHWC [n][h][w][c],
//   except a pooling layer that feeds a fully connected layer (NCHW, the order it reads);
//   the input of a first convolution: NHWC in the compute type (converted from the caller's NCHW);
//   fully connected inputs: the producing layer's layout ((h, w, c) order after a spatial layer);
//   weights as the GEMMs read them (prepared every step from the fp32 master copy):
//     convolution forward        Wf [co][u][v][ci]           (ci = channel within the group)
//     convolution data gradient  Wd [g][ci][u][v][co]        (implicit GEMM)
//                            or  Wc [g][u][v][ci][co]        (col + col2im)
//     fully connected            W  [o][i], with i in (h, w, c) order after a spatial layer;
//   gradients: fp32 in the logical parameter order ([co][ci][u][v], [o][(c, h, w)], bias).
#pragma once

#include <hip/hip_runtime.h>
#include <cstddef>
#include <cstdint>

namespace mtx {

enum Dt { DT_F32 = 0, DT_BF16 = 1 };

// Division by an invariant divisor d (1 <= d < 2^31) for dividends below 2^31:
// q = (umulhi(n, m) + n) >> s with s = ceil(log2 d), m = floor(2^32 (2^s - d) / d) + 1.
struct FastDiv {
    unsigned m, s;
};
FastDiv make_fastdiv(unsigned d);

// Geometry of one convolution.
struct ConvGeom {
    int N;            // images in the launch (whole batch for fwd/dgrad, one shard for wgrad)
    int C, H, W;      // input
    int OC, OH, OW;   // output
    int K, S, PD, G;  // kernel, stride, padding, groups
};

constexpr int kMaxTab = 2048;  // largest LDS index table (entries of 8 bytes, 16 KB)

// Implicit-GEMM arguments.  Each operation (see igemm.h) reads the fields it needs.
struct GemmArgs {
    const void* a;         // activation-like operand (x, dy)
    const void* b;         // weights, or the second activation operand of a weight gradient
    void* out;             // output (activation, data gradient, col, or fp32 gradient rows)
    const float* bias;     // forward: fp32 bias
    const void* mask;      // data gradient: the previous layer's stored output (ReLU mask)
    float* partial;        // split reduction: fp32 partial sums [z][q][p]
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
    int vec_out;           // epilogue rows of 4 outputs (and of the mask) are 16-byte aligned
    int perm_c, perm_hw;   // fully connected weight gradient after a spatial layer: its input
                           // is in (h, w, c) order with perm_c channels and perm_hw positions
    unsigned a_bytes;      // size of tensor a in bytes (buffer-load range)
    unsigned b_bytes;      // size of tensor b in bytes
    int Hp, Wp, Cp, RUN;   // first-layer convolution over a padded input (see conv_fwd_run)
    // weight gradient fused with the average + update (FcWgradUpd): the model's w, v (null
    // for plain SGD) and grad_avg, indexed like a gradient row, and the step's lr and momentum
    float* upd_w;
    float* upd_v;
    float* upd_avg;
    float upd_lr, upd_mu;
    FastDiv fd_ohw, fd_ow, fd_hw, fd_w, fd_c;
    FastDiv fd_run;
    FastDiv fd_kcg, fd_cg, fd_kog, fd_og;  // K*cg, cg, K*og, og (index tables)
};

// GEMM view of one operation: P output rows, Q output columns, K reduction length, Z blocks
// along blockIdx.z before reduction splits (groups x shards), kmax the largest reduction chunk
// one block may take (0: no limit).
struct GemmDims {
    int P, Q, K, Z, kmax;
};
// Launch shape: 32*FP x 32*FQ output tile, BK reduction tile, reduction splits of kchunk.
struct GemmPlan {
    int FP, FQ, BK, splits, kchunk;
};
GemmPlan plan_for(int dt, const GemmDims& d);
size_t partial_elems(int dt, const GemmDims& d);  // fp32 partial sums a launch needs (0 if none)
GemmDims conv_fwd_dims(int dt, const ConvGeom& g);
GemmDims conv_dgrad_dims(int dt, const ConvGeom& g);
GemmDims conv_wgrad_dims(int dt, const ConvGeom& g, int R);
GemmDims conv_dgrad_col_dims(int dt, const ConvGeom& g);
size_t conv_dgrad_col_elems(const ConvGeom& g);
bool conv_dgrad_use_col(const ConvGeom& g);  // data gradient through col + col2im
GemmDims fc_fwd_dims(int dt, int B, int IN, int OUT);
GemmDims fc_dgrad_dims(int dt, int B, int IN, int OUT);
GemmDims fc_wgrad_dims(int dt, int Nb, int R, int IN, int OUT);
int vec_elems(int dt);  // elements per 16-byte load

// `partial` is fp32 scratch of at least partial_elems() elements (may be null when 0).
// x, y: NHWC.  wf: Wf.  y_f32: store fp32 (always in fp32 mode).
hipError_t conv_fwd(Dt dt, const ConvGeom& g, const void* x, const void* wf, const float* bias,
                    void* y, bool y_f32, bool relu, float* partial, hipStream_t s);
// dy, dx: NHWC.  wd: Wd.
hipError_t conv_dgrad(Dt dt, const ConvGeom& g, const void* dy, const void* wd, void* dx,
                      const void* mask, bool mask_f32, float* partial, hipStream_t s);
// Data gradient through an fp32 col buffer of conv_dgrad_col_elems() elements; wc: Wc.
hipError_t conv_dgrad_col(Dt dt, const ConvGeom& g, const void* dy, const void* wc, void* dx,
                          const void* mask, bool mask_f32, float* col,
                          float* partial, hipStream_t s);
// Weight and bias gradient of R shards of g.N images each; x and dy point at the first shard.
hipError_t conv_wgrad(Dt dt, const ConvGeom& g, int R, const void* x, const void* dy,
                      float* grads, long long ld, long long w_off, long long b_off,
                      float* partial, hipStream_t s);
// First-layer convolution (groups 1) over the padded input X'[n][Hp][Wp][Cp]: a zero border of
// PD around the image, Cp >= C channels (the extra ones zero), so that the K*Cp inputs of one
// kernel row are contiguous.  The reduction runs over k = (u, j) with j < RUN (K*Cp rounded up
// to the vector width); the prepared weights Wr[co][u][j] are zero where j does not stand for a
// real (v, ci).  RunGeom holds the padded sizes.
struct RunGeom {
    int Hp, Wp, Cp, RUN;
};
GemmDims conv_fwd_run_dims(int dt, const ConvGeom& g, const RunGeom& r);
GemmDims conv_wgrad_run_dims(int dt, const ConvGeom& g, const RunGeom& r, int R);
hipError_t conv_fwd_run(Dt dt, const ConvGeom& g, const RunGeom& r, const void* xp,
                        const void* wr, const float* bias, void* y, bool y_f32, bool relu,
                        float* partial, hipStream_t s);
hipError_t conv_wgrad_run(Dt dt, const ConvGeom& g, const RunGeom& r, int R, const void* xp,
                          const void* dy, float* grads, long long ld, long long w_off,
                          long long b_off, float* partial, hipStream_t s);
hipError_t fc_fwd(Dt dt, int B, int IN, int OUT, const void* x, const void* w, const float* bias,
                  void* y, bool y_f32, bool relu, float* partial, hipStream_t s);
hipError_t fc_dgrad(Dt dt, int B, int IN, int OUT, const void* dy, const void* w, void* dx,
                    const void* mask, bool mask_f32, float* partial, hipStream_t s);
// perm_c, perm_hw: see GemmArgs (1, 1 when the input is in logical order).
hipError_t fc_wgrad(Dt dt, int Nb, int R, int IN, int OUT, int perm_c, int perm_hw,
                    const void* x, const void* dy, float* grads, long long ld, long long w_off,
                    long long b_off, float* partial, hipStream_t s);
// The fully connected weight gradient of all R shards fused with the average + update of the
// layer's parameters (w, v: null or ignored when mu == 0, avg; indexed like a gradient row);
// fc_wgrad_update_ok tells whether the layer's plan allows it (an unsplit reduction).
bool fc_wgrad_update_ok(Dt dt, int Nb, int R, int IN, int OUT);
hipError_t fc_wgrad_update(Dt dt, int Nb, int R, int IN, int OUT, int perm_c, int perm_hw,
                           const void* x, const void* dy, float* grads, long long ld,
                           long long w_off, long long b_off, float* w, float* v, float* avg,
                           float lr, float mu, hipStream_t s);

// Kernel timing (api.hip): a launcher that enqueues several kernels for one operation calls
// this between them; with timing on, the kernels before and after are timed as separate sites
// (the later one named <site>_<part>).  No effect otherwise.
void timing_split(hipStream_t s, const char* part);
// Launch record (api.hip): every matrix launch reports its shape to the model whose step is
// being enqueued (mtx_get_launches).  flags: kGemmInterleaved, kGemmDirectLds, kGemmFusedUpdate.
constexpr int kGemmInterleaved = 1;  // the interleaved scheduling order of igemm_kernel
constexpr int kGemmDirectLds = 2;    // an operand loaded straight into LDS (igemm_direct_kernel)
constexpr int kGemmFusedUpdate = 4;  // the weight gradient fused with the average + update
void note_gemm(int fp, int fq, int bk, int splits, int flags);

// elementwise.hip

// Weight preparation: one launch converts the fp32 master weights into every layout above.
enum PrepKind {
    PREP_CAST = 0,   // dst[i] = src[i]
    PREP_CONV_F,     // Wf from W[co][ci][u][v]
    PREP_CONV_D,     // Wd
    PREP_CONV_C,     // Wc
    PREP_FC_PERM,    // W[o][(c, h, w)] -> W[o][(h, w, c)]
    PREP_CONV_RUN,   // Wr[co][u][j] of a first-layer convolution over a padded input
};
struct PrepJob {
    int kind;
    int n;             // elements
    long long src;     // element offset in the fp32 weights
    long long dst;     // element offset in the prepared buffer
    int g, cg, og, KK; // convolution: groups, channels per group in / out, K*K
    int C, HW, IN;     // fully connected permutation; C, Cp, K, RUN of a padded first layer
    int Cp, K, RUN;
    int block0;        // first block of this job in the launch
    FastDiv f0, f1, f2;
};
// jobs: device array of njobs entries, blocks = total blocks (sum over jobs).
hipError_t prep_weights(Dt dt, const PrepJob* jobs, int njobs, int blocks, const float* w,
                        void* dst, hipStream_t s);
int prep_blocks(int n);  // blocks one job of n elements takes
void prep_fill_divisors(PrepJob& j);

// NCHW fp32 -> NHWC compute type (C == 1 or H*W == 1: a plain copy / cast).
hipError_t to_nhwc(Dt dt, const float* x, void* dst, int N, int C, int HW, hipStream_t s);
// NCHW fp32 -> the padded input X'[n][PD + h][PD + w][c] of conv_fwd_run (interior channels
// c < C only; the border and the extra channels are never written and must be zero).
hipError_t to_nhwc_padded(Dt dt, const float* x, void* dst, int N, int C, int H, int W,
                          int PD, const RunGeom& r, hipStream_t s);
hipError_t cast_bf16(const float* src, void* dst, size_t n, hipStream_t s);
// Max pooling over NHWC tensors; argmax holds the window position (u*K + v) per output.  The
// pooled tensor (and argmax) is NCHW when out_nchw / dy_nchw is set.
hipError_t pool_fwd(Dt dt, int N, int C, int H, int W, int K, int S, bool out_nchw,
                    const void* x, void* y, uint8_t* argmax, hipStream_t s);
// Max-pool backward.  gate: the pooled output (same layout as dy) when the pooled tensor is a
// ReLU output, else null; a window whose pooled output is not positive passes no gradient, which
// applies the ReLU mask of the layer below.
hipError_t pool_bwd(Dt dt, int N, int C, int H, int W, int K, int S, bool dy_nchw,
                    const uint8_t* argmax, const void* dy, void* dx, const void* gate,
                    hipStream_t s);
// Softmax cross-entropy of B rows; with loss_out set, also the batch-mean loss (block_sums holds
// ceil(B/4) floats; *sync must be 0 before the first launch and is 0 again after every launch).
hipError_t softmax_xent(Dt dt, int B, int NC, int Nb, const float* logits,
                        const int32_t* labels, void* dz, float* block_sums, unsigned* sync,
                        float* loss_out, hipStream_t s);
// max_blocks > 0 caps the grid (the kernel strides over the range), so that an update running
// beside other kernels occupies only part of the GPU.  nonfinite (average only, update false):
// set to 1 when an average is not finite; skip (update): the launch does nothing while *skip.
hipError_t average_update(const float* grads, int R, size_t n, size_t ld, float* w, float* v,
                          float lr, float mu, float* avg, bool update, hipStream_t s,
                          unsigned max_blocks = 0, const int* skip = nullptr,
                          int* nonfinite = nullptr);
// *p = value, as a kernel (graph-capturable, unlike a memset node)
hipError_t set_flag(int* p, int value, hipStream_t s);

// Parameters of the adaptive updates after the average (Adam: s1 = first moment m, s2 =
// second moment v; AdaGrad: s1 = accumulated squared gradients, s2 unused).  c1 = 1 - b1,
// c2 = 1 - b2, ib1 = 1 / (1 - b1^t), ib2 = 1 / (1 - b2^t).  avg (nullable) receives the average.
struct AdaptParams {
    float* w;
    float* s1;
    float* s2;
    float* avg;
    float lr, b1, c1, b2, c2, ib1, ib2, eps;
};
// max_blocks > 0 caps the grid as for average_update.
hipError_t average_adapt(const float* grads, int R, size_t n, size_t ld, bool adam,
                         const AdaptParams& p, hipStream_t s, unsigned max_blocks = 0);

// norm.hip: batch normalisation with per-shard statistics and the residual addition, over
// NHWC tensors [R*Nb][HW][C] of all R shards.
constexpr double kBnEps = 1e-3;
// double partial sums one BN launch needs (the `part` scratch of bn_fwd / bn_bwd)
size_t bn_partial_doubles(Dt dt, int R, int C, int Nb, int HW);
constexpr int kBnStatFloats = 4;  // per (shard, channel): mean, 1/std, gamma/std, beta
// y = gamma (x - mean) / sqrt(var + eps) + beta (ReLU) with the statistics of each shard; stats
// receives [R][4][C] floats (mean, 1 / sqrt(var + eps), gamma / sqrt(var + eps), beta) for the
// apply pass and the backward pass.  C must be at most 256, or a multiple of 16 / element size
// up to 256 such vectors.
// skip (nullable): the residual addition that follows, z = y + skip (relu2: then ReLU), in the
// same pass over y
hipError_t bn_fwd(Dt dt, int R, int Nb, int HW, int C, const void* x, void* y,
                  const float* gamma, const float* beta, double* part, float* stats, bool relu,
                  hipStream_t s, const void* skip = nullptr, void* z = nullptr,
                  bool relu2 = false);
// gamma / beta gradients of every shard into grads[r * ld + w_off / b_off + c], and (dx != null)
// dx = gamma inv (dy - mean(dy) - xhat mean(dy xhat)) times the ReLU mask of the layer below;
// stats are the forward pass's; coef is [R][3][C] floats of scratch.
hipError_t bn_bwd(Dt dt, int R, int Nb, int HW, int C, const void* x, const void* dy, void* dx,
                  const void* mask, bool mask_f32, const float* stats, double* part,
                  float* coef, float* grads, long long ld, long long w_off, long long b_off,
                  hipStream_t s);
// residual addition: y = a + b (ReLU); backward: dx and skip receive dy (each null to skip it),
// masked by the ReLU of the previous layer / of the source layer; skip_add: dy += skip.
hipError_t add_fwd(Dt dt, size_t n, const void* a, const void* b, void* y, bool relu,
                   hipStream_t s);
hipError_t add_bwd(Dt dt, size_t n, const void* dy, void* dx, const void* mask, bool mask_f32,
                   void* skip, const void* smask, bool smask_f32, hipStream_t s);
// dy += skip where smask (the source's stored output, its ReLU) is positive; null: everywhere
hipError_t skip_add(Dt dt, size_t n, void* dy, const void* skip, const void* smask,
                    bool smask_f32, hipStream_t s);

// firstconv.hip: direct kernels for a first convolution with one input channel, stride 1,
// a 3x3, 5x5 or 7x7 window and at most 32 output channels (a multiple of 4) whose image and
// output gradient fit the LDS of one block.
constexpr int kFirstMaxOC = 32;
constexpr size_t kFirstMaxLds = 64 * 1024;
bool first_conv_direct(const ConvGeom& g, int dt);
// x: the input [N][H][W] (one channel) in the compute type; w: fp32 [OC][K][K]; y NHWC.
// With pool.y set, the max pooling above the layer (window = stride = pool.k, NHWC output of the
// conv output's type) is computed too: pool.y its output, pool.argmax its window positions.
struct FirstPoolFwd {
    void* y = nullptr;
    uint8_t* argmax = nullptr;
    int k = 0;
};
// With prep.blocks > 0 the launch also runs the weight preparation (prep_weights' blocks
// after its own; prep.first is set by the launcher).
struct FirstPrep {
    const PrepJob* jobs = nullptr;
    int njobs = 0, blocks = 0, first = 0;
    const float* w = nullptr;
    void* dst = nullptr;
};
bool first_conv_pool_ok(const ConvGeom& g, int pk);
hipError_t first_conv_fwd(Dt dt, const ConvGeom& g, const void* x, const float* w,
                          const float* bias, void* y, bool y_f32, bool relu, hipStream_t s,
                          const FirstPoolFwd& pool = FirstPoolFwd{},
                          const FirstPrep& prep = FirstPrep{});
// weight and bias gradients of R shards of g.N images; partial holds
// first_conv_partial_floats(g, R) floats of scratch.  With pool.dy set, the layer's output
// gradient is not read from dy but formed from the max pooling above it (window = stride =
// pool.k, NHWC): pool.dy its output gradient, pool.argmax its window positions, pool.gate its
// output when this layer has a ReLU (else null).
struct FirstPool {
    const void* dy = nullptr;
    const uint8_t* argmax = nullptr;
    const void* gate = nullptr;
    int k = 0;
};
size_t first_conv_partial_floats(const ConvGeom& g, int R);
hipError_t first_conv_wgrad(Dt dt, const ConvGeom& g, int R, const void* x, const void* dy,
                            float* partial, float* grads, long long ld, long long w_off,
                            long long b_off, hipStream_t s, const FirstPool& pool = FirstPool{});

// dgrad_fused.hip: fp32 data gradient of a stride-1, ungrouped 3x3 or 5x5 convolution with at
// most 60 output channels whose output has at most 64 positions per image, col tile and col2im
// in one kernel (LDS, no col buffer).  w: the fp32 weights [OC][C][K][K]; dy, dx, mask NHWC.
constexpr size_t kDxMaxLds = 80 * 1024;
bool conv_dgrad_fused_ok(const ConvGeom& g, int dt);
hipError_t conv_dgrad_fused(const ConvGeom& g, const float* dy, const float* w, float* dx,
                            const void* mask, bool mask_f32, hipStream_t s);

}  // namespace mtx
