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
// one thread per 16-byte chunk (8 channels) of a pixel: the first chunk
// holds the three colours, the rest are zeros
__global__ void k_img_to_bf16(const float* img, int64_t npix, int q, bf16_t* out) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= npix * q) return;
  const int64_t p = i / q;
  uint4 v = make_uint4(0u, 0u, 0u, 0u);
  if (i == p * q) {
    v.x = f2bf2(img[p * 3], img[p * 3 + 1]);
    v.y = f2bf2(img[p * 3 + 2], 0.f);
  }
  reinterpret_cast<uint4*>(out)[i] = v;
}
void img_to_bf16(hipStream_t st, const float* img, int64_t npix, int Cp, void* out) {
  PG_CHECK(Cp % 8 == 0 && Cp >= 8 && ((uintptr_t)out & 15) == 0, "img_to_bf16: layout");
  const int q = Cp / 8;
  hipLaunchKernelGGL(k_img_to_bf16, dim3((unsigned)cdiv(npix * q, 256)), dim3(256), 0, st, img, npix, q,
                     (bf16_t*)out);
  PG_LAUNCH_CHECK();
}

// --------------------------------------------------- generator output layer
// a = relu((x - mean) * scale + shift) (per channel), img = tanh(conv3x3(a) / sigma + b),
// all in fp32 on the vector ALUs (three output channels leave nothing for a
// matrix unit to tile).  A block computes a 16-row x 64-column output tile:
// per chunk of 8 channels it stages the haloed input tile, normalised once
// per element, in LDS as [row][channel][column]; each lane then owns one
// column of a 4-row strip (its wave's rows), so every staged value it reads
// feeds up to 4 pixels x 3 outputs.  Weights sit in LDS as [c][27] and are
// read as wave-wide broadcasts.
constexpr int kFR = 16;   // output rows per block (4 waves x 4-row strips)
constexpr int kFC = 64;   // output columns per block (one per lane)
constexpr int kFK = 8;    // channels per staged chunk

__global__ __launch_bounds__(256) void k_ghead_fwd(const bf16_t* __restrict__ x, int B, int H, int W, int C, int Cp,
                                                   const float* __restrict__ mean, const float* __restrict__ scale,
                                                   const float* __restrict__ shift, const float* __restrict__ Wt,
                                                   const float* __restrict__ sigma, const float* __restrict__ bias,
                                                   float* __restrict__ img) {
  __shared__ float L[kFR + 2][kFK][kFC + 2];
  extern __shared__ float4 wsh4[];     // [C][7] float4: the 27 weights of channel c, then padding
  float* wsh = reinterpret_cast<float*>(wsh4);
  for (int i = threadIdx.x; i < 28 * C; i += 256) {
    const int c = i / 28, k = i - c * 28;
    wsh[i] = k < 27 ? Wt[k * C + c] : 0.f;
  }
  const int tiles_w = (W + kFC - 1) / kFC, tiles_h = (H + kFR - 1) / kFR;
  int bid = blockIdx.x;
  const int tw = bid % tiles_w;
  bid /= tiles_w;
  const int th = bid % tiles_h;
  const int b = bid / tiles_h;
  const int h0 = th * kFR, w0 = tw * kFC;
  const int t = threadIdx.x, tx = t & 63;
  const int ty = __builtin_amdgcn_readfirstlane(t >> 6);
  float acc[4][3];
#pragma unroll
  for (int o = 0; o < 4; ++o) acc[o][0] = acc[o][1] = acc[o][2] = 0.f;
  // The haloed tile's raw 8-channel vectors of the next chunk are fetched
  // into registers before the current chunk is computed, so their latency
  // hides behind the FMAs; staging normalises them into LDS.
  constexpr int kNP = ((kFR + 2) * (kFC + 2) + 255) / 256;   // tile positions per thread
  uint4 raw[kNP];
  uint32_t inside = 0;   // bit j: position j lies inside the image
#pragma unroll
  for (int j = 0; j < kNP; ++j) {
    const int idx = t + 256 * j;
    const int r = idx / (kFC + 2), col = idx - r * (kFC + 2);
    const int ih = h0 + r - 1, iw = w0 + col - 1;
    if (idx < (kFR + 2) * (kFC + 2) && (unsigned)ih < (unsigned)H && (unsigned)iw < (unsigned)W) inside |= 1u << j;
  }
  auto fetch = [&](int c0) {
#pragma unroll
    for (int j = 0; j < kNP; ++j) {
      const int idx = t + 256 * j;
      const int r = idx / (kFC + 2), col = idx - r * (kFC + 2);
      raw[j] = (inside >> j) & 1
                   ? *reinterpret_cast<const uint4*>(x + (((int64_t)b * H + h0 + r - 1) * W + w0 + col - 1) * Cp + c0)
                   : make_uint4(0u, 0u, 0u, 0u);
    }
  };
  fetch(0);
  for (int c0 = 0; c0 < C; c0 += kFK) {
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kNP; ++j) {
      const int idx = t + 256 * j;
      if (idx >= (kFR + 2) * (kFC + 2)) break;
      const int r = idx / (kFC + 2), col = idx - r * (kFC + 2);
      float v[8];
      unpack8(raw[j], v);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int c = c0 + e;
        v[e] = ((inside >> j) & 1) && c < C ? fmaxf((v[e] - mean[c]) * scale[c] + shift[c], 0.f) : 0.f;
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) L[r][e][col] = v[e];
    }
    __syncthreads();
    if (c0 + kFK < C) fetch(c0 + kFK);
    const int nk = min(kFK, C - c0);
#pragma unroll
    for (int cc = 0; cc < kFK; ++cc) {
      if (cc >= nk) break;
      float w[28];
#pragma unroll
      for (int q = 0; q < 7; ++q) {
        const float4 f = wsh4[(c0 + cc) * 7 + q];
        w[4 * q] = f.x; w[4 * q + 1] = f.y; w[4 * q + 2] = f.z; w[4 * q + 3] = f.w;
      }
#pragma unroll
      for (int rr = 0; rr < 6; ++rr)
#pragma unroll
        for (int s_ = 0; s_ < 3; ++s_) {
          const float v = L[4 * ty + rr][cc][tx + s_];
#pragma unroll
          for (int o = 0; o < 4; ++o) {
            const int r = rr - o;
            if (r >= 0 && r <= 2) {
#pragma unroll
              for (int co = 0; co < 3; ++co) acc[o][co] = fmaf(v, w[co * 9 + r * 3 + s_], acc[o][co]);
            }
          }
        }
    }
  }
  const float inv = 1.f / *sigma;
  const int ow = w0 + tx;
#pragma unroll
  for (int o = 0; o < 4; ++o) {
    const int oh = h0 + 4 * ty + o;
    if (oh < H && ow < W) {
      const int64_t q = (((int64_t)b * H + oh) * W + ow) * 3;
#pragma unroll
      for (int co = 0; co < 3; ++co) img[q + co] = tanhf(acc[o][co] * inv + bias[co]);
    }
  }
}

// da[p][c] = sum_{tap, co} dt[p - tap][co] * W[co][tap][c] / sigma,
// dt = dimg * (1 - img^2) (dimg has channel stride ldd >= 3).  A block
// computes a 2-row x 64-column tile of pixels, all Cp channels: dt of the
// haloed tile is staged in LDS once ([row][col][4], one 16-byte read per
// position), the weights as [tap*3][Cp] scaled by 1/sigma (zero for
// channels >= C).  A work item is 4 consecutive channels x 4 consecutive
// pixels of a row: 432 FMAs per 18 + 27 LDS reads, one 16-byte store per
// pixel (lanes run over channels, so the stores are contiguous).
constexpr int kDR = 2;     // output rows per block
constexpr int kDC = 64;    // output columns per block

__global__ __launch_bounds__(256) void k_ghead_dgrad(const float* __restrict__ dimg, int ldd,
                                                     const float* __restrict__ img, int B, int H, int W, int C,
                                                     int Cp, const float* __restrict__ Wt,
                                                     const float* __restrict__ sigma, float* __restrict__ da) {
  __shared__ float4 dts[kDR + 2][kDC + 2];
  extern __shared__ float4 wsd4[];    // [27][Cp / 4]
  float* wsd = reinterpret_cast<float*>(wsd4);
  const float inv = 1.f / *sigma;
  for (int i = threadIdx.x; i < 27 * Cp; i += 256) {
    const int k = i / Cp, c = i - k * Cp;
    wsd[i] = c < C ? Wt[k * C + c] * inv : 0.f;
  }
  const int tiles_w = (W + kDC - 1) / kDC, tiles_h = (H + kDR - 1) / kDR;
  int bid = blockIdx.x;
  const int tw = bid % tiles_w;
  bid /= tiles_w;
  const int th = bid % tiles_h;
  const int b = bid / tiles_h;
  const int h0 = th * kDR, w0 = tw * kDC;
  for (int idx = threadIdx.x; idx < (kDR + 2) * (kDC + 2); idx += 256) {
    const int r = idx / (kDC + 2), col = idx - r * (kDC + 2);
    const int oh = h0 + r - 1, ow = w0 + col - 1;
    float4 d = make_float4(0.f, 0.f, 0.f, 0.f);
    if ((unsigned)oh < (unsigned)H && (unsigned)ow < (unsigned)W) {
      const int64_t q = ((int64_t)b * H + oh) * W + ow;
      const float y0 = img[q * 3], y1 = img[q * 3 + 1], y2 = img[q * 3 + 2];
      d.x = dimg[q * ldd] * (1.f - y0 * y0);
      d.y = dimg[q * ldd + 1] * (1.f - y1 * y1);
      d.z = dimg[q * ldd + 2] * (1.f - y2 * y2);
    }
    dts[r][col] = d;
  }
  __syncthreads();
  const int ncg = Cp >> 2;
  const int items = ncg * kDR * (kDC / 4);
  for (int it = threadIdx.x; it < items; it += 256) {
    const int cg = it % ncg, pq = it / ncg;
    const int rr = pq / (kDC / 4), cq = pq - rr * (kDC / 4);
    const int oh = h0 + rr, ow0 = w0 + 4 * cq;
    if (oh >= H || ow0 >= W) continue;
    float acc[4][4];
#pragma unroll
    for (int p = 0; p < 4; ++p)
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[p][e] = 0.f;
    // output pixel (oh, ow0 + p) takes dt at (oh - r + 1, ow0 + p - s + 1) =
    // staged position (rr + 2 - r, 4 cq + p + 2 - s)
#pragma unroll
    for (int r = 0; r < 3; ++r) {
      float4 d[6];
#pragma unroll
      for (int j = 0; j < 6; ++j) d[j] = dts[rr + 2 - r][4 * cq + j];
#pragma unroll
      for (int s_ = 0; s_ < 3; ++s_)
#pragma unroll
        for (int co = 0; co < 3; ++co) {
          const float4 wv = wsd4[(co * 9 + r * 3 + s_) * ncg + cg];
#pragma unroll
          for (int p = 0; p < 4; ++p) {
            const float4 dd = d[p + 2 - s_];
            const float dv = co == 0 ? dd.x : (co == 1 ? dd.y : dd.z);
            acc[p][0] = fmaf(dv, wv.x, acc[p][0]);
            acc[p][1] = fmaf(dv, wv.y, acc[p][1]);
            acc[p][2] = fmaf(dv, wv.z, acc[p][2]);
            acc[p][3] = fmaf(dv, wv.w, acc[p][3]);
          }
        }
    }
    const int64_t q0 = ((int64_t)b * H + oh) * W + ow0;
#pragma unroll
    for (int p = 0; p < 4; ++p)
      *reinterpret_cast<float4*>(da + (q0 + p) * Cp + 4 * cg) = make_float4(acc[p][0], acc[p][1], acc[p][2], acc[p][3]);
  }
}

// Weight gradient of the output layer:
//   dW[co][r][s][c] = sum_p dt[p][co] a[p + (r - 1, s - 1)][c],  db[co] = sum_p dt[p][co],
// with a = relu(bn(x)) recomputed from x and dt = dimg (1 - img^2).  A
// block takes kWR output rows of one image; a thread owns 4 channels and
// walks whole rows (rows strip, strip + S, ... of the block), sliding a
// 3x3 window of a (4 channels per position) in registers: one new column
// of 3 loads per pixel feeds 108 FMAs.  The S strips then combine in a
// fixed order through LDS, one output channel at a time, into the block's
// partial; blocks are summed in order by k_ghead_fin.
constexpr int kWR = 16;    // output rows per block

__global__ __launch_bounds__(256) void k_ghead_wgrad(const float* __restrict__ dimg, int ldd,
                                                     const float* __restrict__ img, const bf16_t* __restrict__ x,
                                                     int B, int H, int W, int C, int Cp,
                                                     const float* __restrict__ mean, const float* __restrict__ scale,
                                                     const float* __restrict__ shift, float* __restrict__ part) {
  extern __shared__ float red[];      // [S][9 * Cp] strip partials of one output channel
  const int ncg = Cp >> 2;
  const int S = 256 / ncg;            // strips (threads beyond S * ncg idle)
  const int tiles_h = (H + kWR - 1) / kWR;
  const int b = blockIdx.x / tiles_h, h0 = (blockIdx.x % tiles_h) * kWR;
  const int h1 = min(H, h0 + kWR);
  const int t = threadIdx.x;
  const int cg = t % ncg, strip = t / ncg;
  const bool active = strip < S;
  const int c = 4 * cg;
  float mu[4], sc[4], sh[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const bool ok = active && c + e < C;
    mu[e] = ok ? mean[c + e] : 0.f;
    sc[e] = ok ? scale[c + e] : 0.f;   // zero scale and shift: a = 0 for padded channels
    sh[e] = ok ? shift[c + e] : 0.f;
  }
  float acc[3][9][4];
#pragma unroll
  for (int co = 0; co < 3; ++co)
#pragma unroll
    for (int k = 0; k < 9; ++k)
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[co][k][e] = 0.f;
  float bsum[3] = {0.f, 0.f, 0.f};
  // a at (row, col) for this thread's 4 channels (zero outside the image)
  auto load_a = [&](int row, int col, float* v) {
    if ((unsigned)row < (unsigned)H && (unsigned)col < (unsigned)W) {
      const uint2 q = *reinterpret_cast<const uint2*>(x + (((int64_t)b * H + row) * W + col) * Cp + c);
      const float f[4] = {__uint_as_float(q.x << 16), __uint_as_float(q.x & 0xffff0000u),
                          __uint_as_float(q.y << 16), __uint_as_float(q.y & 0xffff0000u)};
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = fmaxf((f[e] - mu[e]) * sc[e] + sh[e], 0.f);
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = 0.f;
    }
  };
  if (active) {
    for (int h = h0 + strip; h < h1; h += S) {
      // window columns w-1, w, w+1 of rows h-1, h, h+1
      float win[3][3][4];
#pragma unroll
      for (int r = 0; r < 3; ++r) {
        load_a(h + r - 1, -1, win[r][0]);
        load_a(h + r - 1, 0, win[r][1]);
      }
      for (int w = 0; w < W; ++w) {
#pragma unroll
        for (int r = 0; r < 3; ++r) load_a(h + r - 1, w + 1, win[r][2]);
        const int64_t q = ((int64_t)b * H + h) * W + w;
        float dt[3];
#pragma unroll
        for (int co = 0; co < 3; ++co) {
          const float y = img[q * 3 + co];
          dt[co] = dimg[q * ldd + co] * (1.f - y * y);
          bsum[co] += dt[co];
        }
#pragma unroll
        for (int co = 0; co < 3; ++co)
#pragma unroll
          for (int r = 0; r < 3; ++r)
#pragma unroll
            for (int s_ = 0; s_ < 3; ++s_)
#pragma unroll
              for (int e = 0; e < 4; ++e)
                acc[co][r * 3 + s_][e] = fmaf(dt[co], win[r][s_][e], acc[co][r * 3 + s_][e]);
#pragma unroll
        for (int r = 0; r < 3; ++r)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            win[r][0][e] = win[r][1][e];
            win[r][1][e] = win[r][2][e];
          }
      }
    }
  }
  const int nout = 27 * C + 3;
  float* out = part + (int64_t)blockIdx.x * nout;
#pragma unroll
  for (int co = 0; co < 3; ++co) {
    __syncthreads();
    if (active)
#pragma unroll
      for (int k = 0; k < 9; ++k)
#pragma unroll
        for (int e = 0; e < 4; ++e) red[strip * 9 * Cp + k * Cp + c + e] = acc[co][k][e];
    __syncthreads();
    for (int i = t; i < 9 * C; i += 256) {
      const int k = i / C, cc = i - k * C;
      float v = 0.f;
      for (int j = 0; j < S; ++j) v += red[j * 9 * Cp + k * Cp + cc];
      out[(co * 9 + k) * C + cc] = v;
    }
  }
  // bias: every strip's lane cg == 0 holds its rows' sums
  __syncthreads();
  if (active && cg == 0) {
    red[strip * 3] = bsum[0];
    red[strip * 3 + 1] = bsum[1];
    red[strip * 3 + 2] = bsum[2];
  }
  __syncthreads();
  if (t < 3) {
    float v = 0.f;
    for (int j = 0; j < S; ++j) v += red[j * 3 + t];
    out[27 * C + t] = v;
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

static int64_t ghead_wgrad_blocks(int B, int H) { return (int64_t)B * cdiv(H, kWR); }

size_t ghead_ws_bytes(int B, int H, int C) { return align256((size_t)ghead_wgrad_blocks(B, H) * (27 * C + 3) * 4); }

void ghead_fwd(hipStream_t st, const void* x, int B, int H, int W, int C, int Cp, const float* mean,
               const float* scale, const float* shift, const float* Wt, const float* sigma, const float* bias,
               float* img) {
  const int64_t blocks = (int64_t)B * cdiv(H, kFR) * cdiv(W, kFC);
  PG_CHECK(blocks < (1LL << 31) && Cp % 8 == 0 && C <= Cp && C <= 512, "ghead_fwd: shape");
  hipLaunchKernelGGL(k_ghead_fwd, dim3((unsigned)blocks), dim3(256), 28 * C * sizeof(float), st, (const bf16_t*)x,
                     B, H, W, C, Cp, mean, scale, shift, Wt, sigma, bias, img);
  PG_LAUNCH_CHECK();
}

void ghead_bwd(hipStream_t st, const float* dimg, int ldd, const float* img, const void* x, int B, int H, int W,
               int C, int Cp, const float* mean, const float* scale, const float* shift, const float* Wt,
               const float* sigma, float* da, float* dwsn, float* dbias, void* ws) {
  PG_CHECK(W % 4 == 0 && Cp % 4 == 0 && C <= Cp && Cp <= 1024, "ghead_bwd: shape");
  const int64_t dblocks = (int64_t)B * cdiv(H, kDR) * cdiv(W, kDC);
  PG_CHECK(dblocks < (1LL << 31), "ghead_bwd: shape");
  hipLaunchKernelGGL(k_ghead_dgrad, dim3((unsigned)dblocks), dim3(256), 27 * Cp * sizeof(float), st, dimg, ldd,
                     img, B, H, W, C, Cp, Wt, sigma, da);
  const int nch = (int)ghead_wgrad_blocks(B, H);
  const int S = 256 / (Cp / 4);
  const size_t red_bytes = (size_t)S * 9 * Cp * sizeof(float);
  PG_CHECK(S >= 1 && red_bytes <= 64 * 1024, "ghead_bwd: channels");
  hipLaunchKernelGGL(k_ghead_wgrad, dim3(nch), dim3(256), red_bytes, st, dimg, ldd, img, (const bf16_t*)x, B, H, W,
                     C, Cp, mean, scale, shift, (float*)ws);
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
// D head parameter gradients.  Linear weight dw[c] = sum_b dout[b] hs[b][c]
// (16 waves per 64 channels, every 16th sample each, then the 16 sums in
// wave order) and dbias = sum_b dout[b]; the projection embedding, one block
// per class k: dE[k][c] = sum over the samples b of class k, in order, of
// dout[b] hs[b][c] (zero for a class with no sample).
__global__ __launch_bounds__(1024) void k_dhead_dw(const float* hs, const float* dout, int N, int C, float* dw,
                                                   float* dbias) {
  __shared__ float sh[16][64];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int c = blockIdx.x * 64 + lane;
  float s = 0.f;
  if (c < C)
    for (int b = wv; b < N; b += 16) s = fmaf(dout[b], hs[(int64_t)b * C + c], s);
  sh[wv][lane] = s;
  __syncthreads();
  if (wv == 0 && c < C) {
    float t = 0.f;
    for (int i = 0; i < 16; ++i) t += sh[i][lane];
    dw[c] = t;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    float t = 0.f;
    for (int b = 0; b < N; ++b) t += dout[b];
    dbias[0] = t;
  }
}
__global__ __launch_bounds__(256) void k_dhead_de(const float* hs, const float* dout, const int32_t* y, int N, int C,
                                                  float* dE) {
  __shared__ int ys[1024], list[1024];
  __shared__ int cnt;
  const int k = blockIdx.x;
  for (int b = threadIdx.x; b < N; b += 256) ys[b] = y[b];
  __syncthreads();
  if (threadIdx.x == 0) {
    int n = 0;
    for (int b = 0; b < N; ++b)
      if (ys[b] == k) list[n++] = b;
    cnt = n;
  }
  __syncthreads();
  const int n = cnt;
  for (int c = threadIdx.x; c < C; c += 256) {
    float s = 0.f;
    for (int i = 0; i < n; ++i) s = fmaf(dout[list[i]], hs[(int64_t)list[i] * C + c], s);
    dE[(int64_t)k * C + c] = s;
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
    PG_CHECK(N <= 1024, "dhead: batch of at most 1024");
    hipLaunchKernelGGL(k_dhead_dw, dim3((unsigned)cdiv(C, 64)), dim3(1024), 0, st, hs, dout, N, C, dw, dbias);
    hipLaunchKernelGGL(k_dhead_de, dim3((unsigned)n_classes), dim3(256), 0, st, hs, dout, y, N, C, dE);
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
// h0[b][hw][c] = z_chunk[b] . W[hw*C0 + c] / sigma + bias (bf16; c >= C0
// zero).  A block takes 256 consecutive outputs (hw, c) of 16 samples with
// their weight rows and z chunks staged in LDS (zc <= 32).
constexpr int kZcMax = 32;
__global__ __launch_bounds__(256) void k_glin_fwd(const float* z, int dz, int zc, const float* Wt,
                                                  const float* sigma, const float* bias, int B, int C0, int C0p,
                                                  bf16_t* h0) {
  __shared__ float ws[256][kZcMax + 1], zs[16][kZcMax + 1];
  const int t = threadIdx.x;
  const int o0 = blockIdx.x * 256, b0 = blockIdx.y * 16;
  const int nop = 16 * C0p;
  for (int e = t; e < 256 * zc; e += 256) {
    const int oo = e / zc, j = e - oo * zc;
    const int op = o0 + oo, hw = op / C0p, c = op - hw * C0p;
    ws[oo][j] = op < nop && c < C0 ? Wt[(int64_t)(hw * C0 + c) * zc + j] : 0.f;
  }
  for (int e = t; e < 16 * zc; e += 256) {
    const int bb = e / zc, j = e - bb * zc;
    zs[bb][j] = b0 + bb < B ? z[(int64_t)(b0 + bb) * dz + j] : 0.f;
  }
  __syncthreads();
  const int op = o0 + t;
  if (op >= nop) return;
  const int hw = op / C0p, c = op - hw * C0p;
  const float sg = *sigma;
  for (int bb = 0; bb < 16 && b0 + bb < B; ++bb) {
    float v = 0.f;
    if (c < C0) {
      float acc = 0.f;
      for (int j = 0; j < zc; ++j) acc = fmaf(zs[bb][j], ws[t][j], acc);
      v = acc / sg + bias[hw * C0 + c];
    }
    h0[((int64_t)(b0 + bb) * 16 + hw) * C0p + c] = f2bf(v);
  }
}

// dW[o][j] = sum_b dh0[b][o] z[b][j]  (gradient of W/sigma);  dbias[o] = sum_b dh0[b][o]
// A block takes 64 outputs (one per lane) with 16 waves, wave w summing the
// samples w, w + 16, ... with all zc + 1 sums in registers; the 16 partial
// sums then combine in wave order through LDS, one column at a time.
__global__ __launch_bounds__(1024) void k_glin_bwd(const bf16_t* dh0, const float* z, int dz, int zc, int B, int C0,
                                                   int C0p, float* dW, float* dbias) {
  __shared__ float part[16][64];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int o = blockIdx.x * 64 + lane;
  const int no = 16 * C0;
  const bool on = o < no;
  const int hw = on ? o / C0 : 0, c = on ? o - hw * C0 : 0;
  float acc[kZcMax + 1];
#pragma unroll
  for (int j = 0; j <= kZcMax; ++j) acc[j] = 0.f;
  if (on)
    for (int b = wv; b < B; b += 16) {
      const float g = bf2f(dh0[((int64_t)b * 16 + hw) * C0p + c]);
      const float* zb = z + (int64_t)b * dz;
#pragma unroll
      for (int j = 0; j < kZcMax; ++j)
        if (j < zc) acc[j] = fmaf(g, zb[j], acc[j]);
      acc[kZcMax] += g;
    }
  for (int j = 0; j <= zc; ++j) {
    float v = 0.f;
#pragma unroll
    for (int jj = 0; jj <= kZcMax; ++jj)
      if (jj == (j == zc ? kZcMax : j)) v = acc[jj];
    __syncthreads();
    part[wv][lane] = v;
    __syncthreads();
    if (wv == 0 && on) {
      float t = 0.f;
      for (int i = 0; i < 16; ++i) t += part[i][lane];
      if (j < zc) dW[(int64_t)o * zc + j] = t;
      else dbias[o] = t;
    }
  }
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
  PG_CHECK(zc >= 1 && zc <= kZcMax && (int64_t)B * 16 * C0p < (1LL << 31), "glin: z chunk of 1..32");
  hipLaunchKernelGGL(k_glin_fwd, dim3((unsigned)cdiv(16LL * C0p, 256), (unsigned)cdiv(B, 16)), dim3(256), 0, st, z, dz,
                     zc, Wt, sigma, bias, B, C0, C0p, (bf16_t*)h0);
  PG_LAUNCH_CHECK();
}

void glin_bwd(hipStream_t st, const void* dh0, const float* z, int dz, int zc, int B, int C0, int C0p, float* dW,
              float* dbias) {
  PG_CHECK(zc >= 1 && zc <= kZcMax, "glin: z chunk of 1..32");
  hipLaunchKernelGGL(k_glin_bwd, dim3((unsigned)cdiv(16LL * C0, 64)), dim3(1024), 0, st, (const bf16_t*)dh0, z, dz,
                     zc, B, C0, C0p, dW, dbias);
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
// one element; four per thread through 16-byte accesses where aligned
PG_DEV void adam1(float& p, float g, float& m, float& v, float b1, float b2, float lr_t, float c2, float eps) {
  m = b1 * m + (1.f - b1) * g;
  v = b2 * v + (1.f - b2) * g * g;
  p -= lr_t * m / (sqrtf(v * c2) + eps);
}
__global__ void k_adam(float* p, const float* g, float* m, float* v, int64_t n, float b1, float b2, float lr_t,
                       float c2, float eps) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t n4 = n >> 2;
  if (i < n4) {
    float4 pp = reinterpret_cast<float4*>(p)[i], mm = reinterpret_cast<float4*>(m)[i];
    float4 vv = reinterpret_cast<float4*>(v)[i];
    const float4 gg = reinterpret_cast<const float4*>(g)[i];
    adam1(pp.x, gg.x, mm.x, vv.x, b1, b2, lr_t, c2, eps);
    adam1(pp.y, gg.y, mm.y, vv.y, b1, b2, lr_t, c2, eps);
    adam1(pp.z, gg.z, mm.z, vv.z, b1, b2, lr_t, c2, eps);
    adam1(pp.w, gg.w, mm.w, vv.w, b1, b2, lr_t, c2, eps);
    reinterpret_cast<float4*>(p)[i] = pp;
    reinterpret_cast<float4*>(m)[i] = mm;
    reinterpret_cast<float4*>(v)[i] = vv;
  } else if (i < n4 + (n & 3)) {
    const int64_t j = 4 * n4 + (i - n4);
    adam1(p[j], g[j], m[j], v[j], b1, b2, lr_t, c2, eps);
  }
}

void adam(hipStream_t st, float* p, const float* g, float* m, float* v, int64_t n, float b1, float b2, float lr,
          float eps, int64_t t) {
  if (n <= 0) return;
  PG_CHECK((((uintptr_t)p | (uintptr_t)g | (uintptr_t)m | (uintptr_t)v) & 15) == 0, "adam: 16-byte aligned buffers");
  const double lr_t = (double)lr / (1.0 - std::pow((double)b1, (double)t));
  const double c2 = 1.0 / (1.0 - std::pow((double)b2, (double)t));
  const int64_t threads = (n >> 2) + (n & 3);
  hipLaunchKernelGGL(k_adam, dim3((unsigned)cdiv(threads, 256)), dim3(256), 0, st, p, g, m, v, n, b1, b2,
                     (float)lr_t, (float)c2, eps);
  PG_LAUNCH_CHECK();
}

}  // namespace pg
