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

// ------------------------------------------------ per-channel reductions
// Column sums and batch-norm statistics over the rows (pixels) of an NHWC
// tensor, in two fixed-order levels (bitwise reproducible, no atomics).
// Level 1: a block takes a chunk of rows; a thread owns 8 consecutive
// channels (one 16-byte bf16 load or two fp32 loads per row) of the rows
// ro, ro + P, ... of the chunk, P threads sharing each channel group.  The
// P partials per channel then combine in order through LDS.  Level 2 merges
// the chunks.  Statistics use shifted sums per thread (shift = the thread's
// first value, so the sums stay well conditioned) and Chan's parallel
// variance formula for every merge.
constexpr int kRowsPerThread = 32;

struct RedShape {
  int CC, P, rows_blk;
};
// C: channels reduced (real count); the reduction covers cpad(C) channels
inline RedShape red_shape(int C) {
  RedShape r;
  r.CC = (int)(cpad(C) / 8);
  r.P = std::max(1, 256 / r.CC);
  r.rows_blk = r.P * kRowsPerThread;
  return r;
}

template <typename T>
PG_DEV void load8f(const T* p, float* v);
template <>
PG_DEV void load8f<bf16_t>(const bf16_t* p, float* v) {
  unpack8(*reinterpret_cast<const uint4*>(p), v);
}
template <>
PG_DEV void load8f<float>(const float* p, float* v) {
  const float4 a = *reinterpret_cast<const float4*>(p), b = *reinterpret_cast<const float4*>(p + 4);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}

PG_DEV void chan_merge(double& n, double& mu, double& m2, double nb, double mb, double m2b) {
  if (nb <= 0.0) return;
  const double nn = n + nb;
  const double d = mb - mu;
  mu += d * nb / nn;
  m2 += m2b + d * d * n * nb / nn;
  n = nn;
}

// STATS: pa = chunk mean, pb = chunk M2; else pa = chunk sum.  [chunk][C]
template <typename T, bool STATS>
__global__ __launch_bounds__(256) void k_colred(const T* x, int64_t M, int C, int ldc, RedShape sh, float* pa,
                                                float* pb) {
  __shared__ float s_a[256 * 8], s_b[256 * 8];
  __shared__ int s_n[256];
  const int t = threadIdx.x;
  const int cc = t % sh.CC, ro = t / sh.CC;
  const int64_t r0 = (int64_t)blockIdx.x * sh.rows_blk;
  const int64_t r1 = r0 + sh.rows_blk < M ? r0 + sh.rows_blk : M;
  float sft[8], s1[8], s2[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) sft[e] = s1[e] = s2[e] = 0.f;
  int n = 0;
  if (ro < sh.P) {
    for (int64_t r = r0 + ro; r < r1; r += sh.P) {
      float v[8];
      load8f<T>(x + r * ldc + cc * 8, v);
      if (STATS && n == 0) {
#pragma unroll
        for (int e = 0; e < 8; ++e) sft[e] = v[e];
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float d = v[e] - sft[e];
        s1[e] += d;
        if (STATS) s2[e] = fmaf(d, d, s2[e]);
      }
      ++n;
    }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    if (STATS) {
      const float mu = n ? sft[e] + s1[e] / (float)n : 0.f;
      s_a[t * 8 + e] = mu;
      s_b[t * 8 + e] = n ? s2[e] - s1[e] * (s1[e] / (float)n) : 0.f;
    } else {
      s_a[t * 8 + e] = s1[e];
    }
  }
  s_n[t] = n;
  __syncthreads();
  for (int c = t; c < C; c += 256) {
    const int g = c >> 3, e = c & 7;
    if (STATS) {
      double nn = 0.0, mu = 0.0, m2 = 0.0;
      for (int j = 0; j < sh.P; ++j) {
        const int u = j * sh.CC + g;
        chan_merge(nn, mu, m2, (double)s_n[u], (double)s_a[u * 8 + e], (double)s_b[u * 8 + e]);
      }
      pa[(int64_t)blockIdx.x * C + c] = (float)mu;
      pb[(int64_t)blockIdx.x * C + c] = (float)m2;
    } else {
      float sum = 0.f;
      for (int j = 0; j < sh.P; ++j) sum += s_a[(j * sh.CC + g) * 8 + e];
      pa[(int64_t)blockIdx.x * C + c] = sum;
    }
  }
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

size_t colsum_ws_bytes(int64_t M, int C) {
  return align256((size_t)cdiv(M, red_shape(C).rows_blk) * C * 4);
}

void colsum(hipStream_t st, bool f32, const void* x, int64_t M, int C, int ldc, float scale, float* out,
            void* ws) {
  if (M <= 0) {
    fill(st, out, C, 0.f);
    return;
  }
  const RedShape sh = red_shape(C);
  PG_CHECK(ldc >= cpad(C) && ldc % 8 == 0, "colsum: channel stride");
  const int nch = (int)cdiv(M, sh.rows_blk);
  float* part = (float*)ws;
  if (f32)
    hipLaunchKernelGGL((k_colred<float, false>), dim3(nch), dim3(256), 0, st, (const float*)x, M, C, ldc, sh, part,
                       nullptr);
  else
    hipLaunchKernelGGL((k_colred<bf16_t, false>), dim3(nch), dim3(256), 0, st, (const bf16_t*)x, M, C, ldc, sh,
                       part, nullptr);
  hipLaunchKernelGGL(k_colsum_fin, dim3((unsigned)cdiv(C, 64)), dim3(1024), 0, st, part, nch, C, scale, out);
  PG_LAUNCH_CHECK();
}

// ------------------------------------------------------- batch norm
__global__ __launch_bounds__(1024) void k_bn_fin(const float* pmean, const float* pm2, int nch, int rows_blk,
                                                 int64_t M, int C, float eps, float* mean, float* rstd) {
  __shared__ double sn[16][64], smu[16][64], sm2[16][64];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int c = blockIdx.x * 64 + lane;
  double n = 0.0, mu = 0.0, m2 = 0.0;
  if (c < C)
    for (int j = wv; j < nch; j += 16) {
      const double nb = (double)std::min<int64_t>(rows_blk, M - (int64_t)j * rows_blk);
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

size_t bn_stats_ws_bytes(int64_t M, int C) {
  return 2 * align256((size_t)cdiv(M, red_shape(C).rows_blk) * C * 4);
}

void bn_stats(hipStream_t st, bool f32, const void* x, int64_t M, int C, int ldc, float eps, float* mean,
              float* rstd, void* ws) {
  PG_CHECK(M > 0, "bn_stats: empty batch");
  const RedShape sh = red_shape(C);
  PG_CHECK(ldc >= cpad(C) && ldc % 8 == 0, "bn_stats: channel stride");
  const int nch = (int)cdiv(M, sh.rows_blk);
  float* pmean = (float*)ws;
  float* pm2 = (float*)((char*)ws + align256((size_t)nch * C * 4));
  if (f32)
    hipLaunchKernelGGL((k_colred<float, true>), dim3(nch), dim3(256), 0, st, (const float*)x, M, C, ldc, sh, pmean,
                       pm2);
  else
    hipLaunchKernelGGL((k_colred<bf16_t, true>), dim3(nch), dim3(256), 0, st, (const bf16_t*)x, M, C, ldc, sh,
                       pmean, pm2);
  hipLaunchKernelGGL(k_bn_fin, dim3((unsigned)cdiv(C, 64)), dim3(1024), 0, st, pmean, pm2, nch, sh.rows_blk, M, C,
                     eps, mean, rstd);
  PG_LAUNCH_CHECK();
}

// a = [relu]((x - mean[c]) * scale[b][c] + shift[b][c]) stored in the
// activation type: the BN(+ReLU) operand of the next convolution, computed
// once per element instead of once per filter tap.  Padded channels get 0.
// One thread per (pixel, 8 channels): 16-byte loads and stores.
template <typename T>
PG_DEV void store8f(T* p, const float* v);
template <>
PG_DEV void store8f<bf16_t>(bf16_t* p, const float* v) {
  *reinterpret_cast<uint4*>(p) = pack8(v);
}
template <>
PG_DEV void store8f<float>(float* p, const float* v) {
  *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
  *reinterpret_cast<float4*>(p + 4) = make_float4(v[4], v[5], v[6], v[7]);
}

template <typename T>
__global__ __launch_bounds__(256) void k_bn_apply(const T* x, int64_t n8, int CC, FastDiv fdCC, FastDiv fdHW,
                                                  int C, const float* mean, const float* scale,
                                                  const float* shift, int tab_stride, int relu, T* out) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n8) return;
  const int p = (int)fdiv((uint32_t)i, fdCC);
  const int c0 = ((int)i - p * CC) * 8;
  const int b = (int)fdiv((uint32_t)p, fdHW);
  float v[8], mu[8], sc[8], sh[8];
  load8f<T>(x + i * 8, v);
  const int64_t tb = (int64_t)b * tab_stride;
  load8f<float>(mean + c0, mu);
  load8f<float>(scale + tb + c0, sc);
  load8f<float>(shift + tb + c0, sh);
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    float y = (v[e] - mu[e]) * sc[e] + sh[e];
    if (relu) y = fmaxf(y, 0.f);
    v[e] = c0 + e < C ? y : 0.f;
  }
  store8f<T>(out + i * 8, v);
}

void bn_apply(hipStream_t st, bool f32, const void* x, int64_t M, int HW, int C, int Cp, const float* mean,
              const float* scale, const float* shift, int tab_stride, bool relu, void* out) {
  const int CC = Cp / 8;
  const int64_t n8 = M * CC;
  if (n8 == 0) return;
  PG_CHECK(Cp % 8 == 0 && tab_stride % 8 == 0 && n8 < (1LL << 31), "bn_apply: shape");
  PG_CHECK(((uintptr_t)mean | (uintptr_t)scale | (uintptr_t)shift) % 16 == 0, "bn_apply: table alignment");
  const FastDiv fdCC = make_fastdiv(CC), fdHW = make_fastdiv(HW);
  dim3 g((unsigned)cdiv(n8, 256));
  if (f32)
    hipLaunchKernelGGL(k_bn_apply<float>, g, dim3(256), 0, st, (const float*)x, n8, CC, fdCC, fdHW, C, mean,
                       scale, shift, tab_stride, (int)relu, (float*)out);
  else
    hipLaunchKernelGGL(k_bn_apply<bf16_t>, g, dim3(256), 0, st, (const bf16_t*)x, n8, CC, fdCC, fdHW, C, mean,
                       scale, shift, tab_stride, (int)relu, (bf16_t*)out);
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

// Small fp32 GEMM for the conditional-BN linear maps (B x dc by dc x C and
// their transposes): C[i][j] = sum_k A(i, k) B(k, j) [/ *div] [+ C[i][j]],
// A(i, k) = A[i * sai + k * sak], B(k, j) = B[k * sbk + j * sbj].  32 x 32
// tiles through LDS, k in chunks of 32, fixed summation order.
__global__ __launch_bounds__(256) void k_gemm_small(int M, int N, int K, const float* A, int64_t sai,
                                                    int64_t sak, const float* Bm, int64_t sbk, int64_t sbj,
                                                    float* Cm, int64_t ldc, const float* div, int acc) {
  __shared__ float As[32][33], Bs[32][33];
  const int i0 = blockIdx.y * 32, j0 = blockIdx.x * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  float c[4] = {0.f, 0.f, 0.f, 0.f};
  for (int k0 = 0; k0 < K; k0 += 32) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int r = ty + 8 * q;
      // the lane index runs along whichever dimension is contiguous
      int ai, ak;
      if (sak == 1) { ai = r; ak = tx; } else { ai = tx; ak = r; }
      As[ai][ak] = (i0 + ai < M && k0 + ak < K) ? A[(i0 + ai) * sai + (int64_t)(k0 + ak) * sak] : 0.f;
      int bk, bj;
      if (sbj == 1) { bk = r; bj = tx; } else { bk = tx; bj = r; }
      Bs[bk][bj] = (k0 + bk < K && j0 + bj < N) ? Bm[(int64_t)(k0 + bk) * sbk + (j0 + bj) * sbj] : 0.f;
    }
    __syncthreads();
#pragma unroll 8
    for (int kk = 0; kk < 32; ++kk) {
      const float b = Bs[kk][tx];
#pragma unroll
      for (int q = 0; q < 4; ++q) c[q] = fmaf(As[ty + 8 * q][kk], b, c[q]);
    }
    __syncthreads();
  }
  const int j = j0 + tx;
  if (j >= N) return;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int i = i0 + ty + 8 * q;
    if (i >= M) continue;
    float v = div ? c[q] / *div : c[q];
    if (acc) v += Cm[(int64_t)i * ldc + j];
    Cm[(int64_t)i * ldc + j] = v;
  }
}

static void gemm_small(hipStream_t st, int M, int N, int K, const float* A, int64_t sai, int64_t sak,
                       const float* Bm, int64_t sbk, int64_t sbj, float* Cm, int64_t ldc, const float* div,
                       bool acc) {
  if (M <= 0 || N <= 0) return;
  hipLaunchKernelGGL(k_gemm_small, dim3((unsigned)cdiv(N, 32), (unsigned)cdiv(M, 32)), dim3(256), 0, st, M, N, K,
                     A, sai, sak, Bm, sbk, sbj, Cm, ldc, div, (int)acc);
}

// gain = 1 + gain_raw, scale = gain * rstd; padded channels -> 0
__global__ void k_cbn_fix(int B, int C, int Cp, const float* rstd, float* gain, float* bias, float* scale) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= B * Cp) return;
  const int c = i % Cp;
  if (c < C) {
    const float g = 1.f + gain[i];
    gain[i] = g;
    scale[i] = g * rstd[c];
  } else {
    gain[i] = 0.f;
    bias[i] = 0.f;
    scale[i] = 0.f;
  }
}

void cbn_tables(hipStream_t st, const float* cond, int dc, const float* Wg, const float* Wb,
                const float* sg, const float* sb, const float* gain_p, const float* bias_p,
                const float* rstd, int B, int C, int Cp, float* gain, float* bias, float* scale) {
  if (cond) {
    // gain_raw[b][c] = cond[b] . Wg[c] / sigma_g, bias[b][c] = cond[b] . Wb[c] / sigma_b
    gemm_small(st, B, C, dc, cond, dc, 1, Wg, 1, dc, gain, Cp, sg, false);
    gemm_small(st, B, C, dc, cond, dc, 1, Wb, 1, dc, bias, Cp, sb, false);
    hipLaunchKernelGGL(k_cbn_fix, dim3((unsigned)cdiv((int64_t)B * Cp, 256)), dim3(256), 0, st, B, C, Cp, rstd,
                       gain, bias, scale);
    PG_LAUNCH_CHECK();
    return;
  }
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

// pass 2a, per (sample, channel): s1 = sum of the chunk partials of dz,
// s2 = of dz * xhat (fixed order), written over the first chunk's slot;
// per-sample gain / bias gradients when dg_stride != 0.
__global__ void k_bnb_fin1(float* p1, float* p2, int nch, int B, int C, float* dgain, float* dbias,
                           int dg_stride) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (int64_t)B * C) return;
  const int b = (int)(i / C), c = (int)(i - (int64_t)b * C);
  float s1 = 0.f, s2 = 0.f;
  for (int j = 0; j < nch; ++j) {
    const int64_t o = ((int64_t)b * nch + j) * C + c;
    s1 += p1[o];
    s2 += p2[o];
  }
  const int64_t o0 = (int64_t)b * nch * C + c;
  p1[o0] = s1;
  p2[o0] = s2;
  if (dg_stride) {
    dbias[(int64_t)b * dg_stride + c] = s1;
    dgain[(int64_t)b * dg_stride + c] = s2;
  }
}

// pass 2b, per channel: A = sum_b gain*s1 / N, Bc = sum_b gain*s2 / N (and the
// plain-BN gain / bias gradients sum_b s2, sum_b s1); 16 waves stride the
// samples, combined in order.
__global__ __launch_bounds__(1024) void k_bnb_fin2(const float* p1, const float* p2, int nch, int B, int C,
                                                   const float* gain, int tab_stride, int64_t N, float* dgain,
                                                   float* dbias, float* A, float* Bc, int dg_stride) {
  __shared__ float sh[4][16][64];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int c = blockIdx.x * 64 + lane;
  float a = 0.f, bb = 0.f, ab = 0.f, ag = 0.f;
  if (c < C)
    for (int b = wv; b < B; b += 16) {
      const int64_t o0 = (int64_t)b * nch * C + c;
      const float s1 = p1[o0], s2 = p2[o0];
      const float ga = gain[(int64_t)b * tab_stride + c];
      a = fmaf(ga, s1, a);
      bb = fmaf(ga, s2, bb);
      ab += s1;
      ag += s2;
    }
  sh[0][wv][lane] = a; sh[1][wv][lane] = bb; sh[2][wv][lane] = ab; sh[3][wv][lane] = ag;
  __syncthreads();
  if (wv == 0 && c < C) {
    float t[4] = {0.f, 0.f, 0.f, 0.f};
    for (int w = 0; w < 16; ++w)
      for (int q = 0; q < 4; ++q) t[q] += sh[q][w][lane];
    A[c] = t[0] / (float)N;
    Bc[c] = t[1] / (float)N;
    if (!dg_stride) {
      dbias[c] = t[2];
      dgain[c] = t[3];
    }
  }
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
  hipLaunchKernelGGL(k_bnb_fin1, dim3((unsigned)cdiv((int64_t)B * C, 256)), dim3(256), 0, st, p1, p2, nch, B, C,
                     dgain, dbias, dg_stride);
  hipLaunchKernelGGL(k_bnb_fin2, dim3((unsigned)cdiv(C, 64)), dim3(1024), 0, st, p1, p2, nch, B, C, gain,
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
void cbn_linear_bwd(hipStream_t st, const float* dgb, int B, int C, int Cp, const float* cond, int dc,
                    const float* W, const float* sigma, float* dW, float* dcond, bool accumulate) {
  // dW[c][j] = sum_b dgb[b][c] cond[b][j];  dcond[b][j] (+)= sum_c dgb[b][c] W[c][j] / sigma
  gemm_small(st, C, dc, B, dgb, 1, Cp, cond, dc, 1, dW, dc, nullptr, false);
  gemm_small(st, B, dc, C, dgb, Cp, 1, W, dc, 1, dcond, dc, sigma, accumulate);
  PG_LAUNCH_CHECK();
}

// 2x2 average pool, 8 channels per thread
template <typename T>
__global__ __launch_bounds__(256) void k_avgpool2(const T* x, int64_t n8, int CC, FastDiv fdCC, FastDiv fdWo,
                                                  int Ho, int Wo, T* out) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n8) return;
  const int p = (int)fdiv((uint32_t)i, fdCC);
  const int cc = (int)i - p * CC;
  const int t = (int)fdiv((uint32_t)p, fdWo);
  const int j = p - t * Wo;           // t = b * Ho + i
  const int64_t W2 = 2LL * Wo;
  const int64_t r0 = (2LL * t) * W2 + 2 * j;   // (b, 2i, 2j) as a pixel of the input
  const int64_t Cp = (int64_t)CC * 8;
  float a[8], v[8];
  load8f<T>(x + r0 * Cp + cc * 8, a);
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] = a[e];
  load8f<T>(x + (r0 + 1) * Cp + cc * 8, a);
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] += a[e];
  load8f<T>(x + (r0 + W2) * Cp + cc * 8, a);
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] += a[e];
  load8f<T>(x + (r0 + W2 + 1) * Cp + cc * 8, a);
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] = (v[e] + a[e]) * 0.25f;
  (void)Ho;
  store8f<T>(out + i * 8, v);
}

void avgpool2(hipStream_t st, bool f32, const void* x, int B, int H, int W, int Cp, void* out) {
  PG_CHECK(H % 2 == 0 && W % 2 == 0 && Cp % 8 == 0, "avgpool2: shape");
  const int Ho = H / 2, Wo = W / 2, CC = Cp / 8;
  const int64_t n8 = (int64_t)B * Ho * Wo * CC;
  if (n8 == 0) return;
  PG_CHECK(n8 < (1LL << 31), "avgpool2: size");
  const FastDiv fdCC = make_fastdiv(CC), fdWo = make_fastdiv(Wo);
  dim3 g((unsigned)cdiv(n8, 256));
  if (f32)
    hipLaunchKernelGGL(k_avgpool2<float>, g, dim3(256), 0, st, (const float*)x, n8, CC, fdCC, fdWo, Ho, Wo,
                       (float*)out);
  else
    hipLaunchKernelGGL(k_avgpool2<bf16_t>, g, dim3(256), 0, st, (const bf16_t*)x, n8, CC, fdCC, fdWo, Ho, Wo,
                       (bf16_t*)out);
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
