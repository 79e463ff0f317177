// Launchers of the network-level kernels (heads.hip).
#pragma once
#include <cmath>

#include "misc.hpp"

namespace pg {

// fp32 [N][H][W][3] images -> bf16 [N][H][W][32] 3x3 patches (channel (r*3+s)*3+c)
void img_to_im2col(hipStream_t st, const float* img, int N, int H, int W, void* out);
// its adjoint: fp32 patch gradients [N][H][W][32] -> fp32 image gradient [N][H][W][4]
void im2col_grad(hipStream_t st, const float* dcol, int N, int H, int W, float* dimg);

// generator output layer (fp32): img = tanh(conv3x3(relu(bn(x))) + b)
// Shapes the kernels take: cpad(C) <= 128, W a multiple of 4, and the
// weight-gradient tile (one image row plus a frame) within 64 KB of LDS.
bool ghead_shape_ok(int W, int C);
size_t ghead_ws_bytes(int B, int H, int W, int C);
void ghead_fwd(hipStream_t st, const void* x, int B, int H, int W, int C, int Cp, const float* mean,
               const float* scale, const float* shift, const float* Wt, const float* sigma, const float* bias,
               float* img);
// da: fp32 [B][H][W][Cp] gradient of relu(bn(x)); dwsn: [3][3][3][C] gradient of W/sigma
void ghead_bwd(hipStream_t st, const float* dimg, int ldd, const float* img, const void* x, int B, int H, int W,
               int C, int Cp, const float* mean, const float* scale, const float* shift, const float* Wt,
               const float* sigma, float* da, float* dwsn, float* dbias, void* ws);

// projection-discriminator head (fp32) and hinge loss
void dhead_fwd(hipStream_t st, const void* x, int N, int HW, int C, int Cp, const int32_t* y, const float* w,
               const float* sw, const float* bias, const float* E, const float* se, float* hs, float* out);
void hinge(hipStream_t st, const float* out, int nr, int nf, bool gen, float* dout, float* loss);
// dw == nullptr: input gradient only
void dhead_bwd(hipStream_t st, const void* x, int N, int HW, int C, int Cp, const int32_t* y, const float* dout,
               const float* hs, const float* w, const float* sw, const float* E, const float* se, int n_classes,
               void* dx, float* dw, float* dbias, float* dE);

// generator input
void make_cond(hipStream_t st, const float* shared, int sd, const int32_t* y, const float* z, int dz, int zoff,
               int zc, int B, float* cond);
void glin_fwd(hipStream_t st, const float* z, int dz, int zc, const float* Wt, const float* sigma,
              const float* bias, int B, int C0, int C0p, void* h0);
void glin_bwd(hipStream_t st, const void* dh0, const float* z, int dz, int zc, int B, int C0, int C0p, float* dW,
              float* dbias);
void shared_grad(hipStream_t st, const float* dcond, int dc, const int32_t* y, int B, int n_classes, int sd,
                 float* dshared);

// One optimiser step t (>= 1) over n fp32 parameters: kind 0 Adam, 1 AdaBelief.
void optim_step(hipStream_t st, int kind, float* p, const float* g, float* m, float* v, int64_t n, float b1,
                float b2, float lr, float eps, int64_t t);

}  // namespace pg
