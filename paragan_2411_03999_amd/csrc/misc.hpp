// Launchers of the bandwidth-bound kernels (misc.hip, heads.hip, attention.hip).
#pragma once
#include "ops.hpp"

namespace pg {

// spectral normalisation
size_t sn_ws_bytes(int64_t rows, int64_t cols);
// Grouped forms: up to kSnGroupMax SN weights through one launch per phase
// (the job table travels in the kernel arguments, 2.3 KB at 24 jobs).
constexpr int kSnGroupMax = 24;
struct SnJob {
  const float* W;       // [rows][cols] fp32
  int64_t rows, cols;
  float *u, *v, *sigma; // u updated in place; v, sigma written
  float* u_save;        // optional copy of the final u
};
size_t sn_group_ws_bytes(const SnJob* jobs, int n);
// The library's own SN scratch array (one per device, held until the
// process ends) for callers that cannot allocate.  sn_scratch_init() runs
// with `device` current and returns the array's device address there.
constexpr size_t kSnScratchBytes = (size_t)4 << 20;
void* sn_scratch_init(int device);
void sn_power_iter_group(hipStream_t st, const SnJob* jobs, int n, int n_iter, float eps, void* ws);
// Any number of jobs, in groups of kSnGroupMax; ws holds every job's
// partials (sn_group_ws_bytes of all of them).
void sn_power_iter_all(hipStream_t st, const SnJob* jobs, int n, int n_iter, float eps, void* ws);
// mode: kPackFwd [Np][R][R][Cp]; kPackDgrad [Cp][R][R][Np] flipped taps;
// kPackPool4 [Np][4][4][Cp], the 3x3 filter (R = 3) convolved with the 2x2
// averaging box: the stride-2 filter of conv3x3 followed by avgpool2;
// kPackDgradSum4 [Cp][4][4][Np], the flipped transposed 3x3 filter convolved
// with the 2x2 summing box: the stride-2 filter of the data gradient of
// conv3x3 after a nearest 2x upsample (conv3x3^T, then the upsample's
// adjoint, the 2x2 sum).
// kPackSub [4][Np][2][2][Cp]: per parity (a, b) of the output pixels of a
// 3x3 conv over a nearest 2x upsample, the 2x2 filter on the source whose
// taps sum the 3x3 taps landing on one source pixel (rows r in [0, a] for
// tap 0 and [1 + a, 2] for tap 1, columns likewise);
// kPackSubDgrad [4][Cp][2][2][Np]: the same for the flipped transposed
// filter (the data gradient of conv3x3 through a 2x2 average pool).
// kPackDgradRep4 [Cp][2][2][Np]: the transposed 1x1 filter (R = 1) on all
// four taps of a 2x2 window: the stride-2 filter of a 1x1 data gradient
// taken on the 2x2 sum of its input.
enum PackMode {
  kPackFwd = 0, kPackDgrad = 1, kPackPool4 = 2, kPackDgradSum4 = 3, kPackSub = 4, kPackSubDgrad = 5,
  kPackDgradRep4 = 6
};
struct PackJob {
  const float* W;
  const float* sigma;
  void* dst;
  int Cout, Cin, R, Np, Cp;
  int mode;
  int koff = 0;   // kPackFwd / kPackDgrad: input channel c lands at channel koff + c of dst
};
void pack_group(hipStream_t st, bool f32, const PackJob* jobs, int n);
// any number of jobs, in groups of kSnGroupMax
void pack_all(hipStream_t st, bool f32, const PackJob* jobs, int n);
struct SnBwdJob {
  const float *dwp, *W, *u, *v, *sigma, *scale;
  float* dW;
  int Cout, Cin, R, Cp;
};
// part: kSnbParts floats per job (the fixed-order partials of <dWsn, W>)
constexpr int kSnbParts = 1024;
void sn_bwd_group(hipStream_t st, const SnBwdJob* jobs, int n, float* part);
// dw[n][r][s][c] (3x3) = 1/4 sum_{a,b in {0,1}} dw4[n][r+a][s+b][c]: the gradient
// of a 3x3 filter from that of its pooled stride-2 4x4 form
void fold_pool4_wgrad(hipStream_t st, const float* dw4, int Np, int Cp, float* dw);
// u_save (optional) receives a copy of the final u (kept for the backward).
void sn_power_iter(hipStream_t st, const float* W, int64_t rows, int64_t cols, float* u, float* v,
                   float* sigma, int n_iter, float eps, void* ws, float* u_save = nullptr);
void pack_weight(hipStream_t st, bool f32, const float* W, const float* sigma, int Cout, int Cin,
                 int R, int Np, int Cp, bool dgrad, void* dst);
// dst[c][col_off + n] = W[n][c] / sigma for a 1x1 weight W [Cout][Cin]
void pack_weight_t(hipStream_t st, bool f32, const float* W, const float* sigma, int Cout, int Cin, int Cp,
                   int Np, int ld, int col_off, void* dst);
// dW = (s*dWsn - <s*dWsn, W/sigma> u v^T) / sigma with s = *scale (1 if null).
void sn_bwd(hipStream_t st, const float* dwp, const float* W, const float* u, const float* v,
            const float* sigma, int Cout, int Cin, int R, int Cp, const float* scale, float* dW,
            float* part);

// out[c] = scale * sum_m x[m][c]
size_t colsum_ws_bytes(int64_t M, int C);
void colsum(hipStream_t st, bool f32, const void* x, int64_t M, int C, int ldc, float scale, float* out,
            void* ws);

// batch norm
size_t bn_stats_ws_bytes(int64_t M, int C);
void bn_stats(hipStream_t st, bool f32, const void* x, int64_t M, int C, int ldc, float eps, float* mean,
              float* rstd, void* ws);
// out = [relu]((x - mean) * scale + shift), per-(sample, channel) tables;
// mean has Cp entries and each table row (stride tab_stride) Cp, 16-byte aligned
void bn_apply(hipStream_t st, bool f32, const void* x, int64_t M, int HW, int C, int Cp, const float* mean,
              const float* scale, const float* shift, int tab_stride, bool relu, void* out);
void cbn_tables(hipStream_t st, const float* cond, int dc, const float* Wg, const float* Wb,
                const float* sg, const float* sb, const float* gain_p, const float* bias_p,
                const float* rstd, int B, int C, int Cp, float* gain, float* bias, float* scale);
size_t bn_bwd_ws_bytes(int B, int HW, int C);
void bn_bwd(hipStream_t st, bool f32, const float* g, bool g_up2, const void* x, int B, int H, int W,
            int C, int Cp, const float* mean, const float* rstd, const float* gain, const float* bias,
            int tab_stride, const float* res, void* dx, float* dgain, float* dbias, int dg_stride,
            void* ws);
// ws: cbn_linear_bwd_ws_bytes() of scratch for a split-K dcond (may be null)
constexpr int kLinSplits = 8;
size_t cbn_linear_bwd_ws_bytes(int B, int dc);
void cbn_linear_bwd(hipStream_t st, const float* dgb, int B, int C, int Cp, const float* cond, int dc,
                    const float* W, const float* sigma, float* dW, float* dcond, bool accumulate, float* ws);
void fill(hipStream_t st, float* p, int64_t n, float v);
// out[b][i][j][c] = ((x[2i][2j] + x[2i][2j+1]) + x[2i+1][2j]) + x[2i+1][2j+1]) / 4, in the
// activation type (NHWC, channel stride Cp; H and W even)
void avgpool2(hipStream_t st, bool f32, const void* x, int B, int H, int W, int Cp, void* out);

}  // namespace pg
