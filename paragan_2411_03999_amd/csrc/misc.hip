// Bandwidth-bound kernels: spectral normalisation (power iteration, weight
// packing, backward), batch-norm statistics / affine tables / backward,
// bias-gradient column sums.  All reductions run in a fixed order (no float
// atomics), so results are bitwise reproducible run to run.
#include "misc.hpp"

namespace pg {

// ----------------------------------------------------- block reductions
template <int NT>
PG_DEV float block_sum(float v, float* sh) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) sh[w] = v;
  __syncthreads();
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < NT / 64; ++i) s += sh[i];
  __syncthreads();
  return s;
}
template <int NT>
PG_DEV double block_sum_d(double v, double* sh) {
  v = wave_sum_d(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) sh[w] = v;
  __syncthreads();
  double s = 0.0;
#pragma unroll
  for (int i = 0; i < NT / 64; ++i) s += sh[i];
  __syncthreads();
  return s;
}

// ------------------------------------------------ spectral normalisation
// part[rc][c] = sum_{r in chunk rc} W[r][c] u[r]
__global__ void k_sn_wtu(const float* W, const float* u, int64_t rows, int64_t cols, int rchunk,
                         float* part) {
  const int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t r0 = (int64_t)blockIdx.y * rchunk;
  if (c >= cols) return;
  int64_t r1 = r0 + rchunk;
  if (r1 > rows) r1 = rows;
  float s = 0.f;
  for (int64_t r = r0; r < r1; ++r) s = fmaf(W[r * cols + c], u[r], s);
  part[(int64_t)blockIdx.y * cols + c] = s;
}

// v = t / max(|t|, eps), t[c] = sum over row chunks (in order)
__global__ void k_sn_finish_v(const float* part, int nrc, int64_t cols, float eps, float* v) {
  __shared__ double sh[16];
  double ss = 0.0;
  for (int64_t c = threadIdx.x; c < cols; c += 1024) {
    float t = 0.f;
    for (int j = 0; j < nrc; ++j) t += part[(int64_t)j * cols + c];
    v[c] = t;
    ss += (double)t * t;
  }
  const double tot = block_sum_d<1024>(ss, sh);
  const float inv = 1.f / fmaxf((float)sqrt(tot), eps);
  for (int64_t c = threadIdx.x; c < cols; c += 1024) v[c] = v[c] * inv;
}

// s[r] = W[r] . v   (one wave per row)
__global__ void k_sn_wv(const float* W, const float* v, int64_t rows, int64_t cols, float* s) {
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (r >= rows) return;
  float acc = 0.f;
  for (int64_t c = lane; c < cols; c += 64) acc = fmaf(W[r * cols + c], v[c], acc);
  acc = wave_sum(acc);
  if (lane == 0) s[r] = acc;
}

// u = s / max(|s|, eps); sigma = u . s
__global__ void k_sn_finish_u(const float* s, int64_t rows, float eps, float* u, float* u_save,
                              float* sigma) {
  __shared__ double sh[16];
  double ss = 0.0;
  for (int64_t r = threadIdx.x; r < rows; r += 1024) ss += (double)s[r] * s[r];
  const double tot = block_sum_d<1024>(ss, sh);
  const float inv = 1.f / fmaxf((float)sqrt(tot), eps);
  double sg = 0.0;
  for (int64_t r = threadIdx.x; r < rows; r += 1024) {
    const float un = s[r] * inv;
    u[r] = un;
    if (u_save) u_save[r] = un;
    sg += (double)un * s[r];
  }
  const double sgt = block_sum_d<1024>(sg, sh);
  if (threadIdx.x == 0) *sigma = (float)sgt;
}

static int sn_rchunk(int64_t rows) { return rows > 4096 ? 256 : (rows > 256 ? 64 : 16); }

size_t sn_ws_bytes(int64_t rows, int64_t cols) {
  const int64_t nrc = cdiv(rows, sn_rchunk(rows));
  return align256((size_t)nrc * cols * 4) + align256((size_t)rows * 4);
}

void sn_power_iter(hipStream_t st, const float* W, int64_t rows, int64_t cols, float* u, float* v,
                   float* sigma, int n_iter, float eps, void* ws, float* u_save) {
  const int rc = sn_rchunk(rows);
  const int nrc = (int)cdiv(rows, rc);
  float* part = (float*)ws;
  float* s = (float*)((char*)ws + align256((size_t)nrc * cols * 4));
  for (int it = 0; it < n_iter; ++it) {
    hipLaunchKernelGGL(k_sn_wtu, dim3((unsigned)cdiv(cols, 256), nrc), dim3(256), 0, st, W, u, rows,
                       cols, rc, part);
    hipLaunchKernelGGL(k_sn_finish_v, dim3(1), dim3(1024), 0, st, part, nrc, cols, eps, v);
    hipLaunchKernelGGL(k_sn_wv, dim3((unsigned)cdiv(rows, 4)), dim3(256), 0, st, W, v, rows, cols, s);
    hipLaunchKernelGGL(k_sn_finish_u, dim3(1), dim3(1024), 0, st, s, rows, eps, u,
                       it + 1 == n_iter ? u_save : nullptr, sigma);
  }
  PG_LAUNCH_CHECK();
}

// Pack W/sigma into the conv operand layouts.
//  forward: dst[n][r][s][c]  ([Np][R][R][Cp]),  n < Cout, c < Cin
//  dgrad:   dst[c][r][s][n]  ([Cp][R][R][Np]) = W[n][R-1-r][R-1-s][c]
template <typename T>
__global__ void k_pack(const float* W, const float* sigma, int Cout, int Cin, int R, int Np, int Cp,
                       int dgrad, T* dst) {
  const int64_t total = (int64_t)(dgrad ? Cp : Np) * R * R * (dgrad ? Np : Cp);
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= total) return;
  const float inv_s = 1.f / *sigma;
  float v = 0.f;
  if (!dgrad) {
    const int c = (int)(i % Cp);
    const int64_t t = i / Cp;
    const int tap = (int)(t % (R * R));
    const int n = (int)(t / (R * R));
    if (n < Cout && c < Cin) v = W[((int64_t)n * R * R + tap) * Cin + c] / *sigma;
  } else {
    const int n = (int)(i % Np);
    const int64_t t = i / Np;
    const int tap = (int)(t % (R * R));
    const int c = (int)(t / (R * R));
    const int r = tap / R, s = tap % R;
    const int ftap = (R - 1 - r) * R + (R - 1 - s);
    if (n < Cout && c < Cin) v = W[((int64_t)n * R * R + ftap) * Cin + c] / *sigma;
  }
  (void)inv_s;
  st<T>(dst, i, v);
}

void pack_weight(hipStream_t st, bool f32, const float* W, const float* sigma, int Cout, int Cin,
                 int R, int Np, int Cp, bool dgrad, void* dst) {
  const int64_t total = (int64_t)Np * R * R * Cp;
  dim3 g((unsigned)cdiv(total, 256));
  if (f32)
    hipLaunchKernelGGL(k_pack<float>, g, dim3(256), 0, st, W, sigma, Cout, Cin, R, Np, Cp, (int)dgrad,
                       (float*)dst);
  else
    hipLaunchKernelGGL(k_pack<bf16_t>, g, dim3(256), 0, st, W, sigma, Cout, Cin, R, Np, Cp, (int)dgrad,
                       (bf16_t*)dst);
  PG_LAUNCH_CHECK();
}

// Transposed 1x1 pack into columns [col_off, col_off + Np) of a [Cp][ld]
// matrix: dst[c][col_off + n] = W[n][c] / sigma (zero outside Cout x Cin).
template <typename T>
__global__ void k_pack_t(const float* W, const float* sigma, int Cout, int Cin, int Cp, int Np, int ld,
                         int col_off, T* dst) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (int64_t)Cp * Np) return;
  const int n = (int)(i % Np), c = (int)(i / Np);
  const float v = (n < Cout && c < Cin) ? W[(int64_t)n * Cin + c] / *sigma : 0.f;
  st<T>(dst, (int64_t)c * ld + col_off + n, v);
}

void pack_weight_t(hipStream_t st, bool f32, const float* W, const float* sigma, int Cout, int Cin, int Cp,
                   int Np, int ld, int col_off, void* dst) {
  dim3 g((unsigned)cdiv((int64_t)Cp * Np, 256));
  if (f32)
    hipLaunchKernelGGL(k_pack_t<float>, g, dim3(256), 0, st, W, sigma, Cout, Cin, Cp, Np, ld, col_off,
                       (float*)dst);
  else
    hipLaunchKernelGGL(k_pack_t<bf16_t>, g, dim3(256), 0, st, W, sigma, Cout, Cin, Cp, Np, ld, col_off,
                       (bf16_t*)dst);
  PG_LAUNCH_CHECK();
}

// SN backward.  dwp: dL/d(W/sigma) in the padded forward layout
// [Np][R][R][Cp]; W: master [Cout][R][R][Cin].
//   dW = (dWsn - <dWsn, W/sigma> u v^T) / sigma,  v indexed by (r, s, c).
__global__ void k_sn_dot_part(const float* dwp, const float* W, int Cout, int Cin, int RR, int Cp,
                              float* part) {
  __shared__ float sh[4];
  const int64_t total = (int64_t)Cout * RR * Cin;
  float acc = 0.f;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total; i += (int64_t)gridDim.x * 256) {
    const int c = (int)(i % Cin);
    const int64_t t = i / Cin;
    acc = fmaf(dwp[t * Cp + c], W[i], acc);
  }
  const float s = block_sum<256>(acc, sh);
  if (threadIdx.x == 0) part[blockIdx.x] = s;
}

__global__ void k_sn_bwd_apply(const float* dwp, const float* W, const float* u, const float* v,
                               const float* sigma, const float* part, int nparts, int Cout, int Cin,
                               int RR, int Cp, const float* scale_p, float* dW) {
  __shared__ float dotsh;
  const float extra_scale = scale_p ? *scale_p : 1.f;
  if (threadIdx.x == 0) {
    float d = 0.f;
    for (int j = 0; j < nparts; ++j) d += part[j];
    dotsh = d / *sigma;      // <dWsn, W/sigma>
  }
  __syncthreads();
  const float dot = dotsh * extra_scale;
  const float inv = 1.f / *sigma;
  const int64_t total = (int64_t)Cout * RR * Cin;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= total) return;
  const int c = (int)(i % Cin);
  const int64_t t = i / Cin;        // n * RR + tap
  const int n = (int)(t / RR);
  const int64_t k = i - (int64_t)n * RR * Cin;   // column index (tap, c)
  dW[i] = (extra_scale * dwp[t * Cp + c] - dot * u[n] * v[k]) * inv;
}

void sn_bwd(hipStream_t st, const float* dwp, const float* W, const float* u, const float* v,
            const float* sigma, int Cout, int Cin, int R, int Cp, const float* scale, float* dW,
            float* part /* >= 256 floats */) {
  const int RR = R * R;
  const int64_t total = (int64_t)Cout * RR * Cin;
  const int nparts = (int)std::min<int64_t>(256, cdiv(total, 256));
  hipLaunchKernelGGL(k_sn_dot_part, dim3(nparts), dim3(256), 0, st, dwp, W, Cout, Cin, RR, Cp, part);
  hipLaunchKernelGGL(k_sn_bwd_apply, dim3((unsigned)cdiv(total, 256)), dim3(256), 0, st, dwp, W, u, v,
                     sigma, part, nparts, Cout, Cin, RR, Cp, scale, dW);
  PG_LAUNCH_CHECK();
}

// ------------------------------------------------------ column sums
// Two-level fixed-order reduction over rows.  Level 1: block (chunk of
// kRows rows, 64 channels); its 4 waves take rows r = wave (mod 4), lanes
// are consecutive channels (coalesced), the 4 wave sums combine in order.
// Level 2: one block per 64 channels; 16 waves take chunks j = wave
// (mod 16), combined in order.
constexpr int kRows = 2048;

template <typename T>
__global__ __launch_bounds__(256) void k_colsum_part(const T* x, int64_t M, int C, int ldc, float* part) {
  __shared__ float sh[4][64];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int c = blockIdx.y * 64 + lane;
  const int64_t r0 = (int64_t)blockIdx.x * kRows;
  const int64_t r1 = r0 + kRows < M ? r0 + kRows : M;
  float s = 0.f;
  if (c < C)
    for (int64_t r = r0 + wv; r < r1; r += 4) s += ld<T>(x, r * ldc + c);
  sh[wv][lane] = s;
  __syncthreads();
  if (wv == 0 && c < C) part[(int64_t)blockIdx.x * C + c] = (sh[0][lane] + sh[1][lane]) + (sh[2][lane] + sh[3][lane]);
}

__global__ __launch_bounds__(1024) void k_colsum_fin(const float* part, int nch, int C, float scale, float* out) {
  __shared__ float sh[16][64];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int c = blockIdx.x * 64 + lane;
  float s = 0.f;
  if (c < C)
    for (int j = wv; j < nch; j += 16) s += part[(int64_t)j * C + c];
  sh[wv][lane] = s;
  __syncthreads();
  if (wv == 0 && c < C) {
    float t = 0.f;
    for (int i = 0; i < 16; ++i) t += sh[i][lane];
    out[c] = t * scale;
  }
}

size_t colsum_ws_bytes(int64_t M, int C) { return align256((size_t)cdiv(M, kRows) * C * 4); }

void colsum(hipStream_t st, bool f32, const void* x, int64_t M, int C, int ldc, float scale, float* out,
            void* ws) {
  const int nch = (int)cdiv(M, kRows);
  float* part = (float*)ws;
  dim3 g1(nch, (unsigned)cdiv(C, 64));
  if (f32)
    hipLaunchKernelGGL(k_colsum_part<float>, g1, dim3(256), 0, st, (const float*)x, M, C, ldc, part);
  else
    hipLaunchKernelGGL(k_colsum_part<bf16_t>, g1, dim3(256), 0, st, (const bf16_t*)x, M, C, ldc, part);
  hipLaunchKernelGGL(k_colsum_fin, dim3((unsigned)cdiv(C, 64)), dim3(1024), 0, st, part, nch, C, scale, out);
  PG_LAUNCH_CHECK();
}

// ------------------------------------------------------- batch norm
// Per chunk of kRows rows: mean by a first pass, M2 = sum (x - mean)^2 by a
// second (both fixed-order as in the column sums); chunks merge with Chan's
// formula in fp64, in a fixed order.
template <typename T>
__global__ __launch_bounds__(256) void k_bn_part(const T* x, int64_t M, int C, int ldc, float* pmean, float* pm2) {
  __shared__ float sh[4][64];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int c = blockIdx.y * 64 + lane;
  const int64_t r0 = (int64_t)blockIdx.x * kRows;
  const int64_t r1 = r0 + kRows < M ? r0 + kRows : M;
  float s = 0.f;
  if (c < C)
    for (int64_t r = r0 + wv; r < r1; r += 4) s += ld<T>(x, r * ldc + c);
  sh[wv][lane] = s;
  __syncthreads();
  const float mean = ((sh[0][lane] + sh[1][lane]) + (sh[2][lane] + sh[3][lane])) / (float)(r1 - r0);
  __syncthreads();
  float m2 = 0.f;
  if (c < C)
    for (int64_t r = r0 + wv; r < r1; r += 4) {
      const float d = ld<T>(x, r * ldc + c) - mean;
      m2 = fmaf(d, d, m2);
    }
  sh[wv][lane] = m2;
  __syncthreads();
  if (wv == 0 && c < C) {
    pmean[(int64_t)blockIdx.x * C + c] = mean;
    pm2[(int64_t)blockIdx.x * C + c] = (sh[0][lane] + sh[1][lane]) + (sh[2][lane] + sh[3][lane]);
  }
}

PG_DEV void chan_merge(double& n, double& mu, double& m2, double nb, double mb, double m2b) {
  if (nb <= 0.0) return;
  const double nn = n + nb;
  const double d = mb - mu;
  mu += d * nb / nn;
  m2 += m2b + d * d * n * nb / nn;
  n = nn;
}

__global__ __launch_bounds__(1024) void k_bn_fin(const float* pmean, const float* pm2, int nch, int64_t M, int C,
                                                 float eps, float* mean, float* rstd) {
  __shared__ double sn[16][64], smu[16][64], sm2[16][64];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int c = blockIdx.x * 64 + lane;
  double n = 0.0, mu = 0.0, m2 = 0.0;
  if (c < C)
    for (int j = wv; j < nch; j += 16) {
      const double nb = (double)std::min<int64_t>(kRows, M - (int64_t)j * kRows);
      chan_merge(n, mu, m2, nb, pmean[(int64_t)j * C + c], pm2[(int64_t)j * C + c]);
    }
  sn[wv][lane] = n; smu[wv][lane] = mu; sm2[wv][lane] = m2;
  __syncthreads();
  if (wv == 0 && c < C) {
    double tn = 0.0, tmu = 0.0, tm2 = 0.0;
    for (int i = 0; i < 16; ++i) chan_merge(tn, tmu, tm2, sn[i][lane], smu[i][lane], sm2[i][lane]);
    mean[c] = (float)tmu;
    rstd[c] = (float)(1.0 / sqrt(tm2 / tn + (double)eps));
  }
}

size_t bn_stats_ws_bytes(int64_t M, int C) { return 2 * align256((size_t)cdiv(M, kRows) * C * 4); }

void bn_stats(hipStream_t st, bool f32, const void* x, int64_t M, int C, int ldc, float eps, float* mean,
              float* rstd, void* ws) {
  const int nch = (int)cdiv(M, kRows);
  float* pmean = (float*)ws;
  float* pm2 = (float*)((char*)ws + align256((size_t)nch * C * 4));
  dim3 g1(nch, (unsigned)cdiv(C, 64));
  if (f32)
    hipLaunchKernelGGL(k_bn_part<float>, g1, dim3(256), 0, st, (const float*)x, M, C, ldc, pmean, pm2);
  else
    hipLaunchKernelGGL(k_bn_part<bf16_t>, g1, dim3(256), 0, st, (const bf16_t*)x, M, C, ldc, pmean, pm2);
  hipLaunchKernelGGL(k_bn_fin, dim3((unsigned)cdiv(C, 64)), dim3(1024), 0, st, pmean, pm2, nch, M, C, eps, mean,
                     rstd);
  PG_LAUNCH_CHECK();
}

// a = [relu]((x - mean[c]) * scale[b][c] + shift[b][c]) stored in the
// activation type: the BN(+ReLU) operand of the next convolution, computed
// once per element instead of once per filter tap.  Padded channels get 0.
template <typename T>
__global__ void k_bn_apply(const T* x, int64_t M, int HW, int C, int Cp, const float* mean, const float* scale,
                           const float* shift, int tab_stride, int relu, T* out) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= M * Cp) return;
  const int c = (int)(i % Cp);
  float v = 0.f;
  if (c < C) {
    const int b = (int)((i / Cp) / HW);
    const int64_t t = (int64_t)b * tab_stride + c;
    v = (ld<T>(x, i) - mean[c]) * scale[t] + shift[t];
    if (relu) v = fmaxf(v, 0.f);
  }
  st<T>(out, i, v);
}

void bn_apply(hipStream_t st, bool f32, const void* x, int64_t M, int HW, int C, int Cp, const float* mean,
              const float* scale, const float* shift, int tab_stride, bool relu, void* out) {
  dim3 g((unsigned)cdiv(M * Cp, 256));
  if (f32)
    hipLaunchKernelGGL(k_bn_apply<float>, g, dim3(256), 0, st, (const float*)x, M, HW, C, Cp, mean, scale, shift,
                       tab_stride, (int)relu, (float*)out);
  else
    hipLaunchKernelGGL(k_bn_apply<bf16_t>, g, dim3(256), 0, st, (const bf16_t*)x, M, HW, C, Cp, mean, scale,
                       shift, tab_stride, (int)relu, (bf16_t*)out);
  PG_LAUNCH_CHECK();
}

// Conditional-BN tables for the conv prologue and the backward pass:
//   gain[b][c] = 1 + cond[b] . Wg[c] / sigma_g,  bias[b][c] = cond[b] . Wb[c] / sigma_b
//   scale[b][c] = gain * rstd[c]   (prologue: (x - mean) * scale + bias)
// Padded channels (c >= C) get zeros.  With cond == nullptr the gains and
// biases are per-channel parameters (plain affine BN, B = 1).
__global__ void k_cbn_tables(const float* cond, int dc, const float* Wg, const float* Wb, const float* sg,
                             const float* sb, const float* gain_p, const float* bias_p,
                             const float* rstd, int B, int C, int Cp, float* gain, float* bias,
                             float* scale) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= B * Cp) return;
  const int b = i / Cp, c = i % Cp;
  float g = 0.f, h = 0.f;
  if (c < C) {
    if (cond) {
      float ag = 0.f, ab = 0.f;
      for (int j = 0; j < dc; ++j) {
        const float cj = cond[(int64_t)b * dc + j];
        ag = fmaf(cj, Wg[(int64_t)c * dc + j], ag);
        ab = fmaf(cj, Wb[(int64_t)c * dc + j], ab);
      }
      g = 1.f + ag / *sg;
      h = ab / *sb;
    } else {
      g = gain_p[c];
      h = bias_p[c];
    }
  }
  gain[i] = g;
  bias[i] = h;
  scale[i] = c < C ? g * rstd[c] : 0.f;
}

void cbn_tables(hipStream_t st, const float* cond, int dc, const float* Wg, const float* Wb,
                const float* sg, const float* sb, const float* gain_p, const float* bias_p,
                const float* rstd, int B, int C, int Cp, float* gain, float* bias, float* scale) {
  hipLaunchKernelGGL(k_cbn_tables, dim3((unsigned)cdiv((int64_t)B * Cp, 256)), dim3(256), 0, st, cond, dc,
                     Wg, Wb, sg, sb, gain_p, bias_p, rstd, B, C, Cp, gain, bias, scale);
  PG_LAUNCH_CHECK();
}

// BN backward, pass 1: per (sample, channel) sums over the sample's pixels of
//   dz = g * [bn(x) > 0]  and  dz * xhat,  xhat = (x - mean) * rstd,
// where g is the gradient of ReLU(BN(x)) (fp32; optionally given at 2x
// resolution and summed over 2x2 -- the upsample's adjoint).
template <typename T>
__global__ void k_bnb_reduce(const float* g, int g_up2, const T* x, int HW, int H, int W, int C, int Cp,
                             const float* mean, const float* rstd, const float* gain, const float* bias,
                             int tab_stride, int rows_per, float* p1, float* p2) {
  const int b = blockIdx.y;
  const int r0 = blockIdx.x * rows_per;
  const int r1 = min(r0 + rows_per, HW);
  for (int c = threadIdx.x; c < C; c += blockDim.x) {
    const float mu = mean[c], rs = rstd[c];
    const float ga = gain[(int64_t)b * tab_stride + c], be = bias[(int64_t)b * tab_stride + c];
    float s1 = 0.f, s2 = 0.f;
    for (int r = r0; r < r1; ++r) {
      const int64_t m = (int64_t)b * HW + r;
      const float xh = (ld<T>(x, m * Cp + c) - mu) * rs;
      float gv;
      if (!g_up2) {
        gv = g[m * Cp + c];
      } else {
        const int h = r / W, w = r % W;
        const int64_t base = (((int64_t)b * 2 * H + 2 * h) * 2 * W + 2 * w) * Cp + c;
        gv = (g[base] + g[base + Cp]) + (g[base + (int64_t)2 * W * Cp] + g[base + (int64_t)2 * W * Cp + Cp]);
      }
      const float dz = (ga * xh + be > 0.f) ? gv : 0.f;
      s1 += dz;
      s2 = fmaf(dz, xh, s2);
    }
    const int64_t o = ((int64_t)b * gridDim.x + blockIdx.x) * C + c;
    p1[o] = s1;
    p2[o] = s2;
  }
}

// pass 2: dbias[b][c] = sum dz, dgain[b][c] = sum dz*xhat; per channel
//   A[c] = sum_b gain[b][c] dbias[b][c] / N,  Bc[c] = sum_b gain[b][c] dgain[b][c] / N
__global__ void k_bnb_fin(const float* p1, const float* p2, int nch, int B, int C, const float* gain,
                          int tab_stride, int64_t N, float* dgain, float* dbias, float* A, float* Bc,
                          int dg_stride) {
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (c >= C) return;
  float a = 0.f, bb = 0.f;
  float ag = 0.f, ab = 0.f;   // per-channel totals (plain BN)
  for (int b = 0; b < B; ++b) {
    float s1 = 0.f, s2 = 0.f;
    for (int j = 0; j < nch; ++j) {
      const int64_t o = ((int64_t)b * nch + j) * C + c;
      s1 += p1[o];
      s2 += p2[o];
    }
    const float ga = gain[(int64_t)b * tab_stride + c];
    a = fmaf(ga, s1, a);
    bb = fmaf(ga, s2, bb);
    if (dg_stride) {
      dbias[(int64_t)b * dg_stride + c] = s1;
      dgain[(int64_t)b * dg_stride + c] = s2;
    } else {
      ab += s1;
      ag += s2;
    }
  }
  if (!dg_stride) {
    dbias[c] = ab;
    dgain[c] = ag;
  }
  A[c] = a / (float)N;
  Bc[c] = bb / (float)N;
}

// pass 3: dx = rstd * (gain * dz - A - xhat * Bc) (+ res, at the same pixel)
template <typename T>
__global__ void k_bnb_apply(const float* g, int g_up2, const T* x, int64_t M, int HW, int H, int W, int C,
                            int Cp, const float* mean, const float* rstd, const float* gain,
                            const float* bias, int tab_stride, const float* A, const float* Bc,
                            const float* res, T* dx) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= M * Cp) return;
  const int c = (int)(i % Cp);
  const int64_t m = i / Cp;
  float out = 0.f;
  if (c < C) {
    const int b = (int)(m / HW);
    const int r = (int)(m - (int64_t)b * HW);
    const float xh = (ld<T>(x, i) - mean[c]) * rstd[c];
    const float ga = gain[(int64_t)b * tab_stride + c], be = bias[(int64_t)b * tab_stride + c];
    float gv;
    if (!g_up2) {
      gv = g[i];
    } else {
      const int h = r / W, w = r % W;
      const int64_t base = (((int64_t)b * 2 * H + 2 * h) * 2 * W + 2 * w) * Cp + c;
      gv = (g[base] + g[base + Cp]) + (g[base + (int64_t)2 * W * Cp] + g[base + (int64_t)2 * W * Cp + Cp]);
    }
    const float dz = (ga * xh + be > 0.f) ? gv : 0.f;
    out = rstd[c] * (ga * dz - A[c] - xh * Bc[c]);
    if (res) out += res[i];
  }
  st<T>(dx, i, out);
}

size_t bn_bwd_ws_bytes(int B, int HW, int C) {
  const int rows_per = 1024;
  const int nch = (int)cdiv(HW, rows_per);
  return 2 * align256((size_t)B * nch * C * 4) + 2 * align256((size_t)C * 4);
}

void bn_bwd(hipStream_t st, bool f32, const float* g, bool g_up2, const void* x, int B, int H, int W,
            int C, int Cp, const float* mean, const float* rstd, const float* gain, const float* bias,
            int tab_stride, const float* res, void* dx, float* dgain, float* dbias, int dg_stride,
            void* ws) {
  const int HW = H * W;
  const int rows_per = 1024;
  const int nch = (int)cdiv(HW, rows_per);
  float* p1 = (float*)ws;
  float* p2 = (float*)((char*)p1 + align256((size_t)B * nch * C * 4));
  float* A = (float*)((char*)p2 + align256((size_t)B * nch * C * 4));
  float* Bc = (float*)((char*)A + align256((size_t)C * 4));
  const int nt = C >= 256 ? 256 : (int)cdiv(C, 64) * 64;
  dim3 g1(nch, B);
  if (f32)
    hipLaunchKernelGGL(k_bnb_reduce<float>, g1, dim3(nt), 0, st, g, (int)g_up2, (const float*)x, HW, H, W,
                       C, Cp, mean, rstd, gain, bias, tab_stride, rows_per, p1, p2);
  else
    hipLaunchKernelGGL(k_bnb_reduce<bf16_t>, g1, dim3(nt), 0, st, g, (int)g_up2, (const bf16_t*)x, HW, H,
                       W, C, Cp, mean, rstd, gain, bias, tab_stride, rows_per, p1, p2);
  hipLaunchKernelGGL(k_bnb_fin, dim3((unsigned)cdiv(C, 256)), dim3(256), 0, st, p1, p2, nch, B, C, gain,
                     tab_stride, (int64_t)B * HW, dgain, dbias, A, Bc, dg_stride);
  const int64_t M = (int64_t)B * HW;
  dim3 g3((unsigned)cdiv(M * Cp, 256));
  if (f32)
    hipLaunchKernelGGL(k_bnb_apply<float>, g3, dim3(256), 0, st, g, (int)g_up2, (const float*)x, M, HW, H,
                       W, C, Cp, mean, rstd, gain, bias, tab_stride, A, Bc, res, (float*)dx);
  else
    hipLaunchKernelGGL(k_bnb_apply<bf16_t>, g3, dim3(256), 0, st, g, (int)g_up2, (const bf16_t*)x, M, HW,
                       H, W, C, Cp, mean, rstd, gain, bias, tab_stride, A, Bc, res, (bf16_t*)dx);
  PG_LAUNCH_CHECK();
}

// Linear-map gradients of the conditional BN:
//   dW[c][j] = sum_b dgb[b][c] cond[b][j]   (gradient of W/sigma; SN bwd follows)
//   dcond[b][j] (+)= sum_c dgb[b][c] W[c][j] / sigma
__global__ void k_cbn_lin_dw(const float* dgb, int B, int C, int Cp, const float* cond, int dc,
                             float* dW) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= C * dc) return;
  const int c = i / dc, j = i % dc;
  float s = 0.f;
  for (int b = 0; b < B; ++b) s = fmaf(dgb[(int64_t)b * Cp + c], cond[(int64_t)b * dc + j], s);
  dW[i] = s;
}
__global__ void k_cbn_lin_dcond(const float* dgb, int B, int C, int Cp, const float* W, const float* sigma,
                                int dc, int accumulate, float* dcond) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= B * dc) return;
  const int b = i / dc, j = i % dc;
  float s = 0.f;
  for (int c = 0; c < C; ++c) s = fmaf(dgb[(int64_t)b * Cp + c], W[(int64_t)c * dc + j], s);
  s = s / *sigma;
  dcond[i] = accumulate ? dcond[i] + s : s;
}

void cbn_linear_bwd(hipStream_t st, const float* dgb, int B, int C, int Cp, const float* cond, int dc,
                    const float* W, const float* sigma, float* dW, float* dcond, bool accumulate) {
  hipLaunchKernelGGL(k_cbn_lin_dw, dim3((unsigned)cdiv((int64_t)C * dc, 256)), dim3(256), 0, st, dgb, B, C,
                     Cp, cond, dc, dW);
  hipLaunchKernelGGL(k_cbn_lin_dcond, dim3((unsigned)cdiv((int64_t)B * dc, 256)), dim3(256), 0, st, dgb, B,
                     C, Cp, W, sigma, dc, (int)accumulate, dcond);
  PG_LAUNCH_CHECK();
}

// elementwise helpers
__global__ void k_fill(float* p, int64_t n, float v) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) p[i] = v;
}
void fill(hipStream_t st, float* p, int64_t n, float v) {
  if (n <= 0) return;
  hipLaunchKernelGGL(k_fill, dim3((unsigned)cdiv(n, 256)), dim3(256), 0, st, p, n, v);
  PG_LAUNCH_CHECK();
}

}  // namespace pg
