// Network-level kernels around the residual blocks: the fp32 generator
// output layer (BN -> ReLU -> conv3x3 to 3 channels -> tanh) and its
// backward, the fp32 projection-discriminator head, the hinge loss, the
// generator's input linear map and conditioning vectors, the shared class
// embedding's gradient, image conversion and a fused Adam update.
// The last generator and discriminator layers stay in fp32, as the paper's
// mixed-precision policy prescribes (Design, "System Optimizations").
#include "heads.hpp"

namespace pg {

// fp32 [N][H][W][3] images -> bf16 [N][H][W][Cp] (channels >= 3 zero)
__global__ void k_img_to_bf16(const float* img, int64_t npix, int Cp, bf16_t* out) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= npix * Cp) return;
  const int c = (int)(i % Cp);
  const int64_t p = i / Cp;
  out[i] = c < 3 ? f2bf(img[p * 3 + c]) : (bf16_t)0;
}
void img_to_bf16(hipStream_t st, const float* img, int64_t npix, int Cp, void* out) {
  hipLaunchKernelGGL(k_img_to_bf16, dim3((unsigned)cdiv(npix * Cp, 256)), dim3(256), 0, st, img, npix, Cp,
                     (bf16_t*)out);
  PG_LAUNCH_CHECK();
}

// --------------------------------------------------- generator output layer
// a = relu((x - mean) * scale + shift) (per channel), img = tanh(conv3x3(a) / sigma + b),
// all in fp32.  A block computes 128 pixels of one image row: per chunk of
// 32 channels it stages the three input rows it needs, already normalised,
// in LDS (each element transformed once), then each thread accumulates one
// pixel over half of the chunk's channels with the weights read as
// wave-uniform scalars; the two halves combine in a fixed order.
constexpr int kHT = 128;
constexpr int kHC = 32;

__global__ __launch_bounds__(256) void k_ghead_fwd(const bf16_t* __restrict__ x, int B, int H, int W, int C, int Cp,
                                                   const float* __restrict__ mean, const float* __restrict__ scale,
                                                   const float* __restrict__ shift, const float* __restrict__ Wt,
                                                   const float* sigma, const float* __restrict__ bias,
                                                   float* img) {
  __shared__ float As[3][kHT + 2][kHC + 1];
  __shared__ float red[kHT][3];
  __shared__ float tab[3][kHC];
  const int tiles_w = (W + kHT - 1) / kHT;
  const int bid = blockIdx.x;
  const int tw = bid % tiles_w;
  const int bh = bid / tiles_w;
  const int h = bh % H, b = bh / H;
  const int w0 = tw * kHT;
  const int t = threadIdx.x, p = t & (kHT - 1);
  const int half = __builtin_amdgcn_readfirstlane(t >> 7);
  float acc[3] = {0.f, 0.f, 0.f};
  for (int c0 = 0; c0 < C; c0 += kHC) {
    __syncthreads();
    if (t < kHC) {
      const int c = c0 + t;
      tab[0][t] = c < C ? mean[c] : 0.f;
      tab[1][t] = c < C ? scale[c] : 0.f;
      tab[2][t] = c < C ? shift[c] : 0.f;
    }
    __syncthreads();
    for (int idx = t; idx < 3 * (kHT + 2) * 4; idx += 256) {
      const int q = idx & 3;
      const int pix = (idx >> 2) % (kHT + 2);
      const int r = (idx >> 2) / (kHT + 2);
      const int ih = h + r - 1, iw = w0 + pix - 1;
      float v[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = 0.f;
      if (ih >= 0 && ih < H && iw >= 0 && iw < W) {
        unpack8(*reinterpret_cast<const uint4*>(x + (((int64_t)b * H + ih) * W + iw) * Cp + c0 + q * 8), v);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int cl = q * 8 + e;
          v[e] = c0 + cl < C ? fmaxf((v[e] - tab[0][cl]) * tab[1][cl] + tab[2][cl], 0.f) : 0.f;
        }
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) As[r][pix][q * 8 + e] = v[e];
    }
    __syncthreads();
    const int cb = c0 + half * 16;
    if (cb + 16 <= C) {
#pragma unroll
      for (int r = 0; r < 3; ++r)
#pragma unroll
        for (int s_ = 0; s_ < 3; ++s_) {
          const float* wr = Wt + (r * 3 + s_) * C + cb;
          float av[16];
#pragma unroll
          for (int cc = 0; cc < 16; ++cc) av[cc] = As[r][p + s_][half * 16 + cc];
#pragma unroll
          for (int cc = 0; cc < 16; ++cc) {
            acc[0] = fmaf(av[cc], wr[cc], acc[0]);
            acc[1] = fmaf(av[cc], wr[9 * C + cc], acc[1]);
            acc[2] = fmaf(av[cc], wr[18 * C + cc], acc[2]);
          }
        }
    } else {
      const int nc = max(0, C - cb);
      for (int r = 0; r < 3; ++r)
        for (int s_ = 0; s_ < 3; ++s_) {
          const float* wr = Wt + (r * 3 + s_) * C + cb;
          for (int cc = 0; cc < nc; ++cc) {
            const float av = As[r][p + s_][half * 16 + cc];
            acc[0] = fmaf(av, wr[cc], acc[0]);
            acc[1] = fmaf(av, wr[9 * C + cc], acc[1]);
            acc[2] = fmaf(av, wr[18 * C + cc], acc[2]);
          }
        }
    }
  }
  if (half == 1) {
    red[p][0] = acc[0];
    red[p][1] = acc[1];
    red[p][2] = acc[2];
  }
  __syncthreads();
  if (half == 0 && w0 + p < W) {
    const float inv = 1.f / *sigma;
    const int64_t o = (((int64_t)b * H + h) * W + w0 + p) * 3;
#pragma unroll
    for (int co = 0; co < 3; ++co) img[o + co] = tanhf((acc[co] + red[p][co]) * inv + bias[co]);
  }
}

// da[p][c] = sum_{tap, co} dt[p - tap][co] * W[co][tap][c] / sigma,
// dt = dimg * (1 - img^2).   dimg has channel stride ldd (>= 3).
__global__ __launch_bounds__(256) void k_ghead_dgrad(const float* dimg, int ldd, const float* img, int B, int H,
                                                     int W, int C, int Cp, const float* Wt, const float* sigma,
                                                     float* da) {
  extern __shared__ float sw[];
  const int n = 27 * C;
  const float inv = 1.f / *sigma;
  for (int i = threadIdx.x; i < n; i += 256) sw[i] = Wt[i] * inv;
  __syncthreads();
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (int64_t)B * H * W * Cp) return;
  const int c = (int)(i % Cp);
  const int64_t p = i / Cp;
  if (c >= C) { da[i] = 0.f; return; }
  const int w = (int)(p % W);
  const int64_t t = p / W;
  const int h = (int)(t % H);
  const int b = (int)(t / H);
  float s_ = 0.f;
  for (int r = 0; r < 3; ++r) {
    const int oh = h - r + 1;
    if (oh < 0 || oh >= H) continue;
    for (int s = 0; s < 3; ++s) {
      const int ow = w - s + 1;
      if (ow < 0 || ow >= W) continue;
      const int64_t q = ((int64_t)b * H + oh) * W + ow;
      for (int co = 0; co < 3; ++co) {
        const float y = img[q * 3 + co];
        const float dt = dimg[q * ldd + co] * (1.f - y * y);
        s_ = fmaf(dt, sw[(co * 9 + r * 3 + s) * C + c], s_);
      }
    }
  }
  da[i] = s_;
}

// Weight gradient of the output layer.  Per chunk of kHeadRows pixels:
//   part[chunk][co][tap][c] = sum_p dt[p][co] a[p + tap][c],
//   part[chunk][27C + co]   = sum_p dt[p][co]          (bias),
// with dt = dimg (1 - img^2) staged in LDS; a thread owns (tap, c) pairs
// (consecutive c across lanes: coalesced loads of x).  Chunks are then
// summed in a fixed order.
constexpr int kHeadRows = 512;

__global__ __launch_bounds__(256) void k_ghead_wgrad(const float* dimg, int ldd, const float* img, const bf16_t* x,
                                                     int B, int H, int W, int C, int Cp, const float* mean,
                                                     const float* scale, const float* shift, float* part) {
  __shared__ float sdt[kHeadRows][3];
  const int64_t M = (int64_t)B * H * W;
  const int64_t p0 = (int64_t)blockIdx.x * kHeadRows;
  const int np = (int)(p0 + kHeadRows < M ? kHeadRows : M - p0);
  const int nout = 27 * C + 3;
  for (int i = threadIdx.x; i < np; i += 256) {
    const int64_t p = p0 + i;
    for (int co = 0; co < 3; ++co) {
      const float y = img[p * 3 + co];
      sdt[i][co] = dimg[p * ldd + co] * (1.f - y * y);
    }
  }
  __syncthreads();
  float* out = part + (int64_t)blockIdx.x * nout;
  if (threadIdx.x < 3) {
    float sb = 0.f;
    for (int i = 0; i < np; ++i) sb += sdt[i][threadIdx.x];
    out[27 * C + threadIdx.x] = sb;
  }
  const int w00 = (int)(p0 % W);
  const int64_t t0 = p0 / W;
  const int h00 = (int)(t0 % H);
  const int b00 = (int)(t0 / H);
  for (int k = threadIdx.x; k < 9 * C; k += 256) {
    const int c = k % C, tap = k / C;
    const int r = tap / 3, s_ = tap % 3;
    const float mu = mean[c], sc = scale[c], sh = shift[c];
    float a0 = 0.f, a1 = 0.f, a2 = 0.f;
    int b = b00, h = h00, w = w00;
    for (int i = 0; i < np; ++i) {
      const int ih = h + r - 1, iw = w + s_ - 1;
      if (ih >= 0 && ih < H && iw >= 0 && iw < W) {
        const float a = fmaxf((bf2f(x[(((int64_t)b * H + ih) * W + iw) * Cp + c]) - mu) * sc + sh, 0.f);
        a0 = fmaf(sdt[i][0], a, a0);
        a1 = fmaf(sdt[i][1], a, a1);
        a2 = fmaf(sdt[i][2], a, a2);
      }
      if (++w == W) {
        w = 0;
        if (++h == H) { h = 0; ++b; }
      }
    }
    out[(0 * 9 + tap) * C + c] = a0;
    out[(1 * 9 + tap) * C + c] = a1;
    out[(2 * 9 + tap) * C + c] = a2;
  }
}

// fixed-order sum of the chunk partials; the last 3 entries are the bias
__global__ __launch_bounds__(1024) void k_ghead_fin(const float* part, int nch, int n, float* dw, float* dbias) {
  __shared__ float sh[16][64];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int o = blockIdx.x * 64 + lane;
  float s = 0.f;
  if (o < n)
    for (int j = wv; j < nch; j += 16) s += part[(int64_t)j * n + o];
  sh[wv][lane] = s;
  __syncthreads();
  if (wv == 0 && o < n) {
    float t = 0.f;
    for (int i = 0; i < 16; ++i) t += sh[i][lane];
    if (o < n - 3) dw[o] = t;
    else dbias[o - (n - 3)] = t;
  }
}

size_t ghead_ws_bytes(int64_t M, int C) { return align256((size_t)cdiv(M, kHeadRows) * (27 * C + 3) * 4); }

void ghead_fwd(hipStream_t st, const void* x, int B, int H, int W, int C, int Cp, const float* mean,
               const float* scale, const float* shift, const float* Wt, const float* sigma, const float* bias,
               float* img) {
  const int64_t blocks = (int64_t)B * H * cdiv(W, kHT);
  PG_CHECK(blocks < (1LL << 31) && Cp % 8 == 0, "ghead_fwd: shape");
  hipLaunchKernelGGL(k_ghead_fwd, dim3((unsigned)blocks), dim3(256), 0, st, (const bf16_t*)x, B, H, W, C, Cp, mean,
                     scale, shift, Wt, sigma, bias, img);
  PG_LAUNCH_CHECK();
}

void ghead_bwd(hipStream_t st, const float* dimg, int ldd, const float* img, const void* x, int B, int H, int W,
               int C, int Cp, const float* mean, const float* scale, const float* shift, const float* Wt,
               const float* sigma, float* da, float* dwsn, float* dbias, void* ws) {
  const int64_t M = (int64_t)B * H * W;
  hipLaunchKernelGGL(k_ghead_dgrad, dim3((unsigned)cdiv(M * Cp, 256)), dim3(256), 27 * C * sizeof(float), st,
                     dimg, ldd, img, B, H, W, C, Cp, Wt, sigma, da);
  const int nch = (int)cdiv(M, kHeadRows);
  hipLaunchKernelGGL(k_ghead_wgrad, dim3(nch), dim3(256), 0, st, dimg, ldd, img, (const bf16_t*)x, B, H, W, C, Cp,
                     mean, scale, shift, (float*)ws);
  hipLaunchKernelGGL(k_ghead_fin, dim3((unsigned)cdiv(27 * C + 3, 64)), dim3(1024), 0, st, (const float*)ws, nch,
                     27 * C + 3, dwsn, dbias);
  PG_LAUNCH_CHECK();
}

// --------------------------------------------------- discriminator head
// hs[b][c] = sum_hw relu(x[b][hw][c]);
// out[b] = hs[b] . (w / sw) + bias + hs[b] . (E[y_b] / se)
__global__ void k_dhead_fwd(const bf16_t* x, int HW, int C, int Cp, const int32_t* y, const float* w,
                            const float* sw, const float* bias, const float* E, const float* se, float* hs,
                            float* out) {
  __shared__ float sh[4];
  const int b = blockIdx.x;
  const int yb = y[b];
  float part = 0.f;
  for (int c = threadIdx.x; c < C; c += 256) {
    float s = 0.f;
    for (int p = 0; p < HW; ++p) s += fmaxf(bf2f(x[((int64_t)b * HW + p) * Cp + c]), 0.f);
    hs[(int64_t)b * C + c] = s;
    part = fmaf(s, w[c] / *sw + E[(int64_t)yb * C + c] / *se, part);
  }
  part = wave_sum(part);
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = part;
  __syncthreads();
  if (threadIdx.x == 0) out[b] = ((sh[0] + sh[1]) + (sh[2] + sh[3])) + bias[0];
}

// Hinge loss.  mode 0 (discriminator): out[0:nr] real, out[nr:nr+nf] fake,
//   L = mean relu(1 - real) + mean relu(1 + fake);  mode 1 (generator):
//   L = -mean(out[0:nf]).  Writes dL/dout (subgradient 0 at the kinks).
__global__ void k_hinge(const float* out, int nr, int nf, int mode, float* dout, float* loss) {
  __shared__ double sh[4];
  double s = 0.0;
  const int n = mode == 0 ? nr + nf : nf;
  for (int i = threadIdx.x; i < n; i += 256) {
    const float v = out[i];
    if (mode == 0) {
      if (i < nr) {
        s += (double)fmaxf(1.f - v, 0.f) / nr;
        dout[i] = v < 1.f ? -1.f / nr : 0.f;
      } else {
        s += (double)fmaxf(1.f + v, 0.f) / nf;
        dout[i] = v > -1.f ? 1.f / nf : 0.f;
      }
    } else {
      s += -(double)v / nf;
      dout[i] = -1.f / nf;
    }
  }
  s = wave_sum_d(s);
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) *loss = (float)((sh[0] + sh[1]) + (sh[2] + sh[3]));
}

// dx[b][hw][c] = dout[b] (w[c]/sw + E[y_b][c]/se) [x > 0]
__global__ void k_dhead_dx(const bf16_t* x, int N, int HW, int C, int Cp, const int32_t* y, const float* dout,
                           const float* w, const float* sw, const float* E, const float* se, bf16_t* dx) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (int64_t)N * HW * Cp) return;
  const int c = (int)(i % Cp);
  const int b = (int)(i / ((int64_t)HW * Cp));
  float v = 0.f;
  if (c < C && bf2f(x[i]) > 0.f) v = dout[b] * (w[c] / *sw + E[(int64_t)y[b] * C + c] / *se);
  dx[i] = f2bf(v);
}

// dw[c] = sum_b dout[b] hs[b][c];  dbias = sum_b dout[b];
// dE[k][c] = sum_{b: y_b = k} dout[b] hs[b][c]
__global__ void k_dhead_dw(const float* hs, const float* dout, const int32_t* y, int N, int C, int n_classes,
                           float* dw, float* dbias, float* dE) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < C) {
    float s = 0.f;
    for (int b = 0; b < N; ++b) s = fmaf(dout[b], hs[(int64_t)b * C + i], s);
    dw[i] = s;
  }
  if (i == 0) {
    float s = 0.f;
    for (int b = 0; b < N; ++b) s += dout[b];
    dbias[0] = s;
  }
  if (i < (int64_t)n_classes * C) {
    const int k = (int)(i / C), c = (int)(i % C);
    float s = 0.f;
    for (int b = 0; b < N; ++b)
      if (y[b] == k) s = fmaf(dout[b], hs[(int64_t)b * C + c], s);
    dE[i] = s;
  }
}

void dhead_fwd(hipStream_t st, const void* x, int N, int HW, int C, int Cp, const int32_t* y, const float* w,
               const float* sw, const float* bias, const float* E, const float* se, float* hs, float* out) {
  hipLaunchKernelGGL(k_dhead_fwd, dim3(N), dim3(256), 0, st, (const bf16_t*)x, HW, C, Cp, y, w, sw, bias, E, se,
                     hs, out);
  PG_LAUNCH_CHECK();
}

void hinge(hipStream_t st, const float* out, int nr, int nf, bool gen, float* dout, float* loss) {
  hipLaunchKernelGGL(k_hinge, dim3(1), dim3(256), 0, st, out, nr, nf, gen ? 1 : 0, dout, loss);
  PG_LAUNCH_CHECK();
}

void dhead_bwd(hipStream_t st, const void* x, int N, int HW, int C, int Cp, const int32_t* y, const float* dout,
               const float* hs, const float* w, const float* sw, const float* E, const float* se, int n_classes,
               void* dx, float* dw, float* dbias, float* dE) {
  hipLaunchKernelGGL(k_dhead_dx, dim3((unsigned)cdiv((int64_t)N * HW * Cp, 256)), dim3(256), 0, st,
                     (const bf16_t*)x, N, HW, C, Cp, y, dout, w, sw, E, se, (bf16_t*)dx);
  if (dw) {
    const int64_t n = std::max<int64_t>((int64_t)n_classes * C, C);
    hipLaunchKernelGGL(k_dhead_dw, dim3((unsigned)cdiv(n, 256)), dim3(256), 0, st, hs, dout, y, N, C, n_classes,
                       dw, dbias, dE);
  }
  PG_LAUNCH_CHECK();
}

// --------------------------------------------------- generator input
// cond[b] = [shared[y_b] (sd) || z[b][zoff : zoff + zc]]
__global__ void k_make_cond(const float* shared, int sd, const int32_t* y, const float* z, int dz, int zoff, int zc,
                            int B, float* cond) {
  const int dc = sd + zc;
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= B * dc) return;
  const int b = i / dc, j = i % dc;
  cond[i] = j < sd ? shared[(int64_t)y[b] * sd + j] : z[(int64_t)b * dz + zoff + j - sd];
}

// h0[b][(h*4+w)][c] = z[b][0:zc] . W[o] / sigma + bias[o],  o = (h*4+w)*C0 + c
__global__ void k_glin_fwd(const float* z, int dz, int zc, const float* Wt, const float* sigma, const float* bias,
                           int B, int C0, int C0p, bf16_t* h0) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (int64_t)B * 16 * C0p) return;
  const int c = (int)(i % C0p);
  const int64_t t = i / C0p;
  const int hw = (int)(t % 16);
  const int b = (int)(t / 16);
  float v = 0.f;
  if (c < C0) {
    const int o = hw * C0 + c;
    float s = 0.f;
    for (int j = 0; j < zc; ++j) s = fmaf(z[(int64_t)b * dz + j], Wt[(int64_t)o * zc + j], s);
    v = s / *sigma + bias[o];
  }
  h0[i] = f2bf(v);
}

// dW[o][j] = sum_b dh0[b][o] z[b][j]  (gradient of W/sigma);  dbias[o] = sum_b dh0[b][o]
__global__ void k_glin_bwd(const bf16_t* dh0, const float* z, int dz, int zc, int B, int C0, int C0p, float* dW,
                           float* dbias) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t no = 16LL * C0;
  if (i >= no * (zc + 1)) return;
  const int64_t o = i / (zc + 1);
  const int j = (int)(i % (zc + 1));
  const int hw = (int)(o / C0), c = (int)(o % C0);
  float s = 0.f;
  for (int b = 0; b < B; ++b) {
    const float g = bf2f(dh0[((int64_t)b * 16 + hw) * C0p + c]);
    s = j < zc ? fmaf(g, z[(int64_t)b * dz + j], s) : s + g;
  }
  if (j < zc) dW[o * zc + j] = s;
  else dbias[o] = s;
}

// dshared[k][d] = sum_{b: y_b = k} dcond[b][d]   (d < sd)
__global__ void k_shared_grad(const float* dcond, int dc, const int32_t* y, int B, int n_classes, int sd,
                              float* dshared) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (int64_t)n_classes * sd) return;
  const int k = (int)(i / sd), d = (int)(i % sd);
  float s = 0.f;
  for (int b = 0; b < B; ++b)
    if (y[b] == k) s += dcond[(int64_t)b * dc + d];
  dshared[i] = s;
}

void make_cond(hipStream_t st, const float* shared, int sd, const int32_t* y, const float* z, int dz, int zoff,
               int zc, int B, float* cond) {
  hipLaunchKernelGGL(k_make_cond, dim3((unsigned)cdiv((int64_t)B * (sd + zc), 256)), dim3(256), 0, st, shared, sd,
                     y, z, dz, zoff, zc, B, cond);
  PG_LAUNCH_CHECK();
}

void glin_fwd(hipStream_t st, const float* z, int dz, int zc, const float* Wt, const float* sigma,
              const float* bias, int B, int C0, int C0p, void* h0) {
  hipLaunchKernelGGL(k_glin_fwd, dim3((unsigned)cdiv((int64_t)B * 16 * C0p, 256)), dim3(256), 0, st, z, dz, zc, Wt,
                     sigma, bias, B, C0, C0p, (bf16_t*)h0);
  PG_LAUNCH_CHECK();
}

void glin_bwd(hipStream_t st, const void* dh0, const float* z, int dz, int zc, int B, int C0, int C0p, float* dW,
              float* dbias) {
  hipLaunchKernelGGL(k_glin_bwd, dim3((unsigned)cdiv(16LL * C0 * (zc + 1), 256)), dim3(256), 0, st,
                     (const bf16_t*)dh0, z, dz, zc, B, C0, C0p, dW, dbias);
  PG_LAUNCH_CHECK();
}

void shared_grad(hipStream_t st, const float* dcond, int dc, const int32_t* y, int B, int n_classes, int sd,
                 float* dshared) {
  hipLaunchKernelGGL(k_shared_grad, dim3((unsigned)cdiv((int64_t)n_classes * sd, 256)), dim3(256), 0, st, dcond, dc,
                     y, B, n_classes, sd, dshared);
  PG_LAUNCH_CHECK();
}

// --------------------------------------------------- Adam
// m = b1 m + (1-b1) g;  v = b2 v + (1-b2) g^2;  p -= lr_t m / (sqrt(v c2) + eps)
// with lr_t = lr / (1 - b1^t) and c2 = 1 / (1 - b2^t) (bias corrections).
__global__ void k_adam(float* p, const float* g, float* m, float* v, int64_t n, float b1, float b2, float lr_t,
                       float c2, float eps) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  const float gi = g[i];
  const float mi = b1 * m[i] + (1.f - b1) * gi;
  const float vi = b2 * v[i] + (1.f - b2) * gi * gi;
  m[i] = mi;
  v[i] = vi;
  p[i] -= lr_t * mi / (sqrtf(vi * c2) + eps);
}

void adam(hipStream_t st, float* p, const float* g, float* m, float* v, int64_t n, float b1, float b2, float lr,
          float eps, int64_t t) {
  const double lr_t = (double)lr / (1.0 - std::pow((double)b1, (double)t));
  const double c2 = 1.0 / (1.0 - std::pow((double)b2, (double)t));
  hipLaunchKernelGGL(k_adam, dim3((unsigned)cdiv(n, 256)), dim3(256), 0, st, p, g, m, v, n, b1, b2, (float)lr_t,
                     (float)c2, eps);
  PG_LAUNCH_CHECK();
}

}  // namespace pg
