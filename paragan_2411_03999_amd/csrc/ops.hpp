// Host-side launchers of the gfx950 kernels.  Every launcher enqueues on the
// given stream and returns immediately; shapes are validated by the callers
// (the C-ABI layer) before anything is launched.
#pragma once
#include "common.hpp"
#include "fastdiv.hpp"

namespace pg {

// Operand gathers of the implicit-GEMM convolutions.  G_S2 reads the
// source at stride 2 (a 4 x 4, pad-1 filter over a source of twice the conv
// grid's size): a 3x3 conv followed by a 2x2 average pool, evaluated at the
// pooled pixels only with the pre-pooled 4 x 4 weights (2.25x fewer MACs);
// with a 2 x 2, pad-0 filter it is a 1x1 conv over the 2x2 sums of the
// source, read once without materialising the sums.
// G_SUB evaluates a 3x3 conv over the nearest 2x upsample of the source as
// four 2x2 convs over the source itself, one per parity class (a, b) of the
// output pixels (2i + a, 2j + b), with the 3x3 taps that fall on the same
// source pixel summed (2.25x fewer MACs); the rows are source-grid pixels,
// blockIdx.y the parity, and the epilogue writes the upsampled position.
enum Gather { G_DIRECT = 0, G_UP2 = 1, G_POOL2 = 2, G_S2 = 3, G_SUB = 4 };
enum ResMode { R_NONE = 0, R_SAME = 1, R_HALF = 2 };

// The A operand of an implicit-GEMM convolution: an NHWC activation read
// through a gather (direct, nearest 2x upsample, or 2x2 sum-pool), scaled,
// optionally batch-normalised with per-(sample, channel) affine tables and
// ReLU'd -- all applied while staging the operand, before the MMA.
struct ConvIn {
  const void* x = nullptr;
  int B = 0, Hx = 0, Wx = 0, C = 0;   // source dims; C = channel stride (x32)
  int gather = G_DIRECT;
  float gscale = 1.f;
  const float* mean = nullptr;        // [C]      (affine prologue)
  const float* scale = nullptr;       // [B][C] or [C]
  const float* shift = nullptr;
  int tab_stride = 0;                 // C for per-sample tables, 0 for per-channel
  int relu = 0;
  int c_real = 0;                     // real input channels (0: = C); for FLOP counts
};

// Epilogue: v = (acc * (*acc_scale) * acc_mul / (*acc_div) + bias[n]) * (mask > 0)
//              + res_scale * res,
// optionally 2x2 average-pooled (the output rows are then the pooled pixels).
// acc_div carries the spectral norm sigma of a filter packed unnormalised.
struct ConvOut {
  void* y = nullptr;
  int y_f32 = 0;
  int yC = 0;                  // channel stride of y
  int n_real = 0;              // channels >= n_real are written as 0
  const float* bias = nullptr;
  const float* acc_scale = nullptr;   // device scalar
  float acc_mul = 1.f;                // host scalar (also multiplies acc)
  const float* acc_div = nullptr;     // device scalar dividing acc (sigma)
  int pool = 0;
  const void* res = nullptr;
  int res_f32 = 0, res_mode = R_NONE, resC = 0;
  float res_scale = 1.f;
  const void* mask = nullptr;         // same position as the output
  int mask_f32 = 0, maskC = 0;
};

// y = conv_RxR(gathered/transformed x, w) on an H x W grid (stride 1, pad R/2).
// w: packed [Np][R][R][in.C] in the activation type (bf16 or fp32).
void conv_fwd(hipStream_t s, bool f32, const ConvIn& in, int H, int W, int R,
              const void* w, int Np, const ConvOut& out);

// The MFMA convolution for direct / upsampled operands without a BN-affine
// prologue (convfwd.hip); conv_fwd dispatches to it when conv_fwd_mfma_ok.
bool conv_fwd_mfma_ok(const ConvIn& in, int H, int W, int R, int Np, const ConvOut& out);
std::string conv_fwd_mfma(hipStream_t s, const ConvIn& in, int H, int W, int R, const void* w, int Np,
                          const ConvOut& out);

// Gradient operand of a weight gradient: dy at the conv-output grid (H x W)
// read directly or as a nearest-2x upsample of a half-resolution tensor.
struct GradIn {
  const void* g = nullptr;
  int Hs = 0, Ws = 0, C = 0;   // source dims; C = channel stride (= Np)
  int gather = G_DIRECT;       // G_DIRECT or G_UP2
  float gscale = 1.f;          // applied to the result
  int n_real = 0;              // real gradient channels (0: = Np); for FLOP counts
};

// dw[n][r][s][c] = gscale * sum_m g[m][n] * A[m][(r,s,c)], A = im2col(in).
// dw: fp32 [Np][R][R][in.C] (padded).  ws: scratch for split-M partials.
size_t conv_wgrad_ws(bool f32, int64_t M, int R, int Cin, int Np, int n_cu);
void conv_wgrad(hipStream_t s, bool f32, const GradIn& g, const ConvIn& in,
                int H, int W, int R, int Np, float* dw, void* ws, size_t ws_bytes,
                int n_cu);

// bf16 weight gradient through LDS transpose reads (wgrad.hip), for direct or
// upsampled operands without a BN-affine prologue.  wgrad_tr_ok tells whether
// a call qualifies; conv_wgrad dispatches to it.
bool wgrad_tr_ok(const GradIn& g, const ConvIn& in, int H, int W, int R, int Np);

// bf16 weight gradient of a 3x3 conv over a nearest 2x upsample of in (the
// source, [B][Hx][Wx][C], direct gather) against g ([B][2 Hx][2 Wx][g.C]),
// through the four sub-pixel 2x2 forms and a fold onto the 3x3 filter:
// dw fp32 [Np][3][3][in.C] = g.gscale * the same sums as conv_wgrad over the
// upsampled operand.  ws: wgrad_sub_ws bytes (per-class partials).
bool wgrad_sub_ok(const GradIn& g, const ConvIn& in, int Np);
size_t wgrad_sub_ws(int64_t Msrc, int Cin, int Np, int n_cu);
void wgrad_sub(hipStream_t s, const GradIn& g, const ConvIn& in, int Np, float* dw, void* ws, size_t ws_bytes,
               int n_cu);
size_t wgrad_tr_ws(int64_t M, int R, int Cin, int Np, int n_cu);
void wgrad_tr(hipStream_t s, const GradIn& g, const ConvIn& in, int H, int W, int R, int Np, float* dw,
              void* ws, size_t ws_bytes, int n_cu, double flops);

}  // namespace pg
