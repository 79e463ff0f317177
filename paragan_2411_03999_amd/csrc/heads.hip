// Network-level kernels around the residual blocks: the fp32 generator
// output layer (BN -> ReLU -> conv3x3 to 3 channels -> tanh) and its
// backward, the fp32 projection-discriminator head, the hinge loss, the
// generator's input linear map and conditioning vectors, the shared class
// embedding's gradient, image conversion and a fused Adam update.
// The last generator and discriminator layers stay in fp32, as the paper's
// mixed-precision policy prescribes (Design, "System Optimizations").
#include "heads.hpp"

namespace pg {

// fp32 [N][H][W][3] images -> bf16 [N][H][W][32] 3x3 patches: channel
// (r * 3 + s) * 3 + c holds img[h + r - 1][w + s - 1][c] (zero outside the
// image), channels 27..31 zero.  The discriminator's first 3x3 conv is then
// a 1x1 conv over 27 real channels instead of 9 taps over 3 of 32.  Both
// this and its adjoint take kPR rows x kPC columns of one image per block:
// the rows it needs, with a one-pixel zero frame, are staged in LDS with
// coalesced loads, then a thread per pixel gathers from LDS.
constexpr int kPR = 2, kPC = 128;

__global__ __launch_bounds__(256) void k_img_im2col(const float* __restrict__ img, int H, int W,
                                                    bf16_t* __restrict__ out) {
  __shared__ float sx[kPR + 2][kPC + 2][3];
  const int ncb = (W + kPC - 1) / kPC, nrb = (H + kPR - 1) / kPR;
  int bid = blockIdx.x;
  const int cb = bid % ncb;
  bid /= ncb;
  const int h0 = (bid % nrb) * kPR, n = bid / nrb, w0 = cb * kPC;
  const float* im = img + (int64_t)n * H * W * 3;
  constexpr int kNS = (kPR + 2) * (kPC + 2) * 3;
#pragma unroll
  for (int k = 0; k < (kNS + 255) / 256; ++k) {
    const int i = threadIdx.x + 256 * k;
    if (i < kNS) {
      const int c = i % 3, q = i / 3, col = q % (kPC + 2), row = q / (kPC + 2);
      const int h = h0 - 1 + row, w = w0 - 1 + col;
      (&sx[0][0][0])[i] =
          (unsigned)h < (unsigned)H && (unsigned)w < (unsigned)W ? im[((int64_t)h * W + w) * 3 + c] : 0.f;
    }
  }
  __syncthreads();
  // 16-byte chunk j of the block's output: pixel j / 4, channels 8 (j % 4) ..;
  // consecutive lanes store consecutive chunks
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int j = threadIdx.x + 256 * k, px = j >> 2, qd = j & 3;
    const int lr = px / kPC, lc = px % kPC;
    const int h = h0 + lr, w = w0 + lc;
    if (h >= H || w >= W) continue;
    float v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int ch = 8 * qd + e, tap = ch / 3, c = ch - 3 * tap;
      v[e] = ch < 27 ? sx[lr + tap / 3][lc + tap % 3][c] : 0.f;
    }
    reinterpret_cast<uint4*>(out + (((int64_t)n * H + h) * W + w) * 32)[qd] = pack8(v);
  }
}
void img_to_im2col(hipStream_t st, const float* img, int N, int H, int W, void* out) {
  PG_CHECK(N >= 1 && H >= 1 && W >= 1 && ((uintptr_t)out & 15) == 0, "img_to_im2col: shape");
  const int64_t blocks = (int64_t)N * cdiv(H, kPR) * cdiv(W, kPC);
  PG_CHECK(blocks < (1LL << 31), "img_to_im2col: too many pixels");
  hipLaunchKernelGGL(k_img_im2col, dim3((unsigned)blocks), dim3(256), 0, st, img, H, W, (bf16_t*)out);
  PG_LAUNCH_CHECK();
}

// The adjoint: dimg[p][c] = sum_{r,s} dcol[p - (r - 1, s - 1)][(r * 3 + s) * 3 + c]
// over the patches that contain p; dcol fp32 [N][H][W][32], dimg fp32
// [N][H][W][4] (channel 3 written as 0).  The staged patch gradients keep
// channels 0..27 (28 floats per pixel: a stride that spreads the lanes of a
// gather over the LDS banks).
constexpr int kPS = 28;
__global__ __launch_bounds__(256) void k_im2col_grad(const float* __restrict__ dcol, int H, int W,
                                                     float* __restrict__ dimg) {
  __shared__ float4 sd[(kPR + 2) * (kPC + 2) * kPS / 4];
  const int ncb = (W + kPC - 1) / kPC, nrb = (H + kPR - 1) / kPR;
  int bid = blockIdx.x;
  const int cb = bid % ncb;
  bid /= ncb;
  const int h0 = (bid % nrb) * kPR, n = bid / nrb, w0 = cb * kPC;
  const float* dc = dcol + (int64_t)n * H * W * 32;
  constexpr int kNS = (kPR + 2) * (kPC + 2) * (kPS / 4);
#pragma unroll
  for (int k = 0; k < (kNS + 255) / 256; ++k) {
    const int i = threadIdx.x + 256 * k;
    if (i < kNS) {
      const int j = i % (kPS / 4), q = i / (kPS / 4), col = q % (kPC + 2), row = q / (kPC + 2);
      const int h = h0 - 1 + row, w = w0 - 1 + col;
      sd[i] = (unsigned)h < (unsigned)H && (unsigned)w < (unsigned)W
                  ? *reinterpret_cast<const float4*>(dc + ((int64_t)h * W + w) * 32 + 4 * j)
                  : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  }
  __syncthreads();
  const int lr = threadIdx.x / kPC, lc = threadIdx.x % kPC;
  const int h = h0 + lr, w = w0 + lc;
  if (h >= H || w >= W) return;
  const float* sf = reinterpret_cast<const float*>(sd);
  float d[3] = {0.f, 0.f, 0.f};
#pragma unroll
  for (int r = 0; r < 3; ++r)
#pragma unroll
    for (int s = 0; s < 3; ++s) {
      // the patch centred at (h - r + 1, w - s + 1) holds this pixel at tap (r, s)
      const float* src = sf + ((lr + 2 - r) * (kPC + 2) + (lc + 2 - s)) * kPS + (r * 3 + s) * 3;
#pragma unroll
      for (int c = 0; c < 3; ++c) d[c] += src[c];
    }
  reinterpret_cast<float4*>(dimg)[((int64_t)n * H + h) * W + w] = make_float4(d[0], d[1], d[2], 0.f);
}
void im2col_grad(hipStream_t st, const float* dcol, int N, int H, int W, float* dimg) {
  PG_CHECK(N >= 1 && H >= 1 && W >= 1 && ((uintptr_t)dimg & 15) == 0 && ((uintptr_t)dcol & 15) == 0,
           "im2col_grad: shape");
  const int64_t blocks = (int64_t)N * cdiv(H, kPR) * cdiv(W, kPC);
  PG_CHECK(blocks < (1LL << 31), "im2col_grad: too many pixels");
  hipLaunchKernelGGL(k_im2col_grad, dim3((unsigned)blocks), dim3(256), 0, st, dcol, H, W, dimg);
  PG_LAUNCH_CHECK();
}

// --------------------------------------------------- generator output layer
// a = relu((x - mean) * scale + shift) per channel; img = tanh(conv3x3(a) / sigma + b).
// Forward and weight gradient run on the fp32 matrix cores
// (v_mfma_f32_32x32x2_f32: fp32 operands and accumulation, so the last layer
// keeps full precision).  The 27 filter columns n = co * 9 + r * 3 + s (27 of
// a 32-wide tile) are the N side of both products; the 3x3 window turns into
// 9-term gathers around them.
constexpr int kHR = 16;     // output rows per forward block
constexpr int kZS = 33;     // LDS floats per Z position (odd: conflict-free gathers)
constexpr int kZP = 130;    // Z positions per ring row: 128 output columns + 2 halo

PG_DEV f32x16 mfma_f32(float a, float b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}
// output columns per forward block: whole rows up to 128, else 126 (so the
// Z columns of a block, its columns plus a halo, fit four 32-position tiles)
static int ghead_cols(int W) { return W <= 128 ? W : 126; }

// Forward.  Z[q][n] = sum_c a[q][c] W[n][c] for every input position q (K =
// the channels, each input value read once), then img[p][co] = tanh(sum_{r,s}
// Z[p + (r - 1, s - 1)][co * 9 + r * 3 + s] / sigma + b[co]).  A block takes
// kHR output rows x ghead_cols(W) output columns of one image and walks its Z
// rows top to bottom: each of the 4 waves computes one 32-position tile of a
// Z row into a 3-row LDS ring (rows outside the image are never read), then
// the block gathers the output row whose three Z rows are present.  A wave
// loads its x values for the next Z row before the current row's products.
// A lane of the product holds position l % 32 and channels 16 j + 8 (l / 32)
// + 0..7 of chunk j: one 16-byte load feeds 8 products.
template <int CK>   // CK = Cp / 16
__global__ __launch_bounds__(256, 2) void k_ghead_fwd(const bf16_t* __restrict__ x, int H, int W, int C, int TC,
                                                      const float* __restrict__ mean, const float* __restrict__ scale,
                                                      const float* __restrict__ shift, const float* __restrict__ Wt,
                                                      const float* __restrict__ sigma, const float* __restrict__ bias,
                                                      float* __restrict__ img) {
  constexpr int Cp = 16 * CK;
  __shared__ float Zs[3][kZP][kZS];
  __shared__ float Wl[CK * 512];          // [j][k][s][n] = W[n][16 j + 8 k + s], zero for n >= 27, c >= C
  __shared__ float4 cst[3][Cp / 4];       // mean, scale, shift (zero for padded channels)
  const int tid = threadIdx.x, lane = tid & 63, kh = lane >> 5, ln = lane & 31;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  for (int i = tid; i < CK * 512; i += 256) {
    const int n = i & 31, s = (i >> 5) & 7, k = (i >> 8) & 1, j = i >> 9;
    const int c = 16 * j + 8 * k + s;
    Wl[i] = n < 27 && c < C ? Wt[n * C + c] : 0.f;
  }
  for (int c = tid; c < Cp; c += 256) {
    const bool ok = c < C;
    reinterpret_cast<float*>(cst[0])[c] = ok ? mean[c] : 0.f;
    reinterpret_cast<float*>(cst[1])[c] = ok ? scale[c] : 0.f;
    reinterpret_cast<float*>(cst[2])[c] = ok ? shift[c] : 0.f;
  }
  const int ncb = (W + TC - 1) / TC, nrb = (H + kHR - 1) / kHR;
  int bid = blockIdx.x;
  const int cb = bid % ncb;
  bid /= ncb;
  const int rb = bid % nrb;
  const int b = bid / nrb;
  const int w0 = cb * TC, h0 = rb * kHR;
  const int w1 = min(W, w0 + TC), h1 = min(H, h0 + kHR);
  const int zc0 = max(0, w0 - 1), zc1 = min(W, w1 + 1);   // Z columns the block needs
  const bool has_tile = 32 * wv < zc1 - zc0;
  const int zw = zc0 + 32 * wv + ln;                        // this lane's Z column
  const bool col_ok = zw < zc1;
  uint4 xr[CK];
  auto fetch = [&](int zr) {
    // columns past zc1 read zeros; their Z values are never gathered
    const bool ok = col_ok && zr >= 0 && zr < H;
    const int64_t off = ok ? (((int64_t)b * H + zr) * W + zw) * Cp + 8 * kh : 0;
#pragma unroll
    for (int j = 0; j < CK; ++j)
      xr[j] = ok ? *reinterpret_cast<const uint4*>(x + off + 16 * j) : make_uint4(0u, 0u, 0u, 0u);
  };
  const float inv = 1.f / *sigma;
  const int nz = h1 - h0 + 2;   // Z rows h0 - 1 .. h1
  fetch(h0 - 1);
  // ring indices 0 and w1 - w0 + 1 are columns w0 - 1 and w1: outside the
  // image (zeros, set once) when the block touches the left or right edge,
  // otherwise written with every Z row
  for (int i = tid; i < 6 * kZS; i += 256) {
    const int side = i / (3 * kZS), k = i - side * 3 * kZS;
    if (side == 0 ? w0 == 0 : w1 == W) Zs[k / kZS][side == 0 ? 0 : w1 - w0 + 1][k % kZS] = 0.f;
  }
  __syncthreads();
  // the B operand of every k-step stays in registers for the whole block
  float wr[CK * 8];
#pragma unroll
  for (int i = 0; i < CK * 8; ++i) wr[i] = Wl[((2 * (i >> 3) + kh) * 8 + (i & 7)) * 32 + ln];
  // BN constants of chunk j for this lane's 8 channels (16 j + 8 kh ..)
  auto ldc = [&](int j, float4 (&c)[6]) {
    const int q4 = 4 * j + 2 * kh;
#pragma unroll
    for (int a = 0; a < 3; ++a) {
      c[2 * a] = cst[a][q4];
      c[2 * a + 1] = cst[a][q4 + 1];
    }
  };
  for (int t = 0; t < nz; ++t) {
    const int zr = h0 - 1 + t;
    uint4 cur[CK];
#pragma unroll
    for (int j = 0; j < CK; ++j) cur[j] = xr[j];
    if (t + 1 < nz) fetch(zr + 1);
    if (has_tile && zr >= 0 && zr < H) {
      f32x16 acc;
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[r] = 0.f;
      float4 cc[6], cn[6];
      ldc(0, cc);
#pragma unroll
      for (int j = 0; j < CK; ++j) {
        if (j + 1 < CK) ldc(j + 1, cn);
        float v[8];
        unpack8(cur[j], v);
        const float mu[8] = {cc[0].x, cc[0].y, cc[0].z, cc[0].w, cc[1].x, cc[1].y, cc[1].z, cc[1].w};
        const float sc[8] = {cc[2].x, cc[2].y, cc[2].z, cc[2].w, cc[3].x, cc[3].y, cc[3].z, cc[3].w};
        const float sh[8] = {cc[4].x, cc[4].y, cc[4].z, cc[4].w, cc[5].x, cc[5].y, cc[5].z, cc[5].w};
#pragma unroll
        for (int s = 0; s < 8; ++s) acc = mfma_f32(fmaxf((v[s] - mu[s]) * sc[s] + sh[s], 0.f), wr[8 * j + s], acc);
#pragma unroll
        for (int i = 0; i < 6; ++i) cc[i] = cn[i];
      }
      // lane: Z[position row 8 (r / 4) + 4 kh + r % 4 of the tile][n = ln].  Ring
      // index w - w0 + 1 stays below kZP for every position of the tiles;
      // columns >= W get zeros (the zero padding the gather reads)
      float* zs = &Zs[t % 3][0][0];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int w = zc0 + 32 * wv + 8 * (r >> 2) + 4 * kh + (r & 3);
        zs[(w - w0 + 1) * kZS + ln] = w < W ? acc[r] : 0.f;
      }
    } else if (zr < 0 || zr >= H) {
      // a Z row outside the image: zeros wherever the gather reads
      float* zs = &Zs[t % 3][0][0];
      for (int i = tid; i < kZP * kZS; i += 256) zs[i] = 0.f;
    }
    if (t >= 2) {
      // output row oh = zr - 1: its Z rows oh - 1 .. oh + 1 sit in ring slots
      // (t - 2 .. t) % 3; every read below lands on a computed or zeroed entry
      __syncthreads();
      const int oh = zr - 1, ncol = w1 - w0;
      const float* z0 = &Zs[(t - 2) % 3][0][0];
      const float* z1 = &Zs[(t - 1) % 3][0][0];
      const float* z2 = &Zs[t % 3][0][0];
      float* const orow = img + (((int64_t)b * H + oh) * W + w0) * 3;
      for (int it = tid; it < 3 * ncol; it += 256) {
        const int pc = it / 3, co = it - 3 * pc;
        const int base = pc * kZS + co * 9;   // ring index of column ow - 1 is pc
        float sum = 0.f;
#pragma unroll
        for (int s = 0; s < 3; ++s) sum += z0[base + s * kZS + s];
#pragma unroll
        for (int s = 0; s < 3; ++s) sum += z1[base + s * kZS + 3 + s];
#pragma unroll
        for (int s = 0; s < 3; ++s) sum += z2[base + s * kZS + 6 + s];
        // tanh(y) = 1 - 2 / (exp(2 y) + 1): exact at the saturated ends,
        // absolute error about 1e-7 elsewhere
        const float e = __expf(2.f * (sum * inv + bias[co]));
        orow[it] = 1.f - __fdividef(2.f, e + 1.f);
      }
      __syncthreads();
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
//   dW[co][r][s][c] = sum_p dt[p][co] a[p + (r - 1, s - 1)][c] = sum_q a[q][c] G[q][n],
//   G[q][co * 9 + r * 3 + s] = dt[q - (r - 1, s - 1)][co],  db[co] = sum_p dt[p][co],
// with a = relu(bn(x)) recomputed from x and dt = dimg (1 - img^2): the
// positions q are the K side of a (C x 32) product on the fp32 matrix cores.
// A block takes ghead_wrows(W) rows of one image.  dt of those rows plus a
// one-pixel zero frame is staged in LDS, so the 27 columns of G are plain
// reads from it; each wave takes 16-position chunks of a, normalised once
// into its LDS tile [position][channel] (the channel is the M side of the
// product).  The 4 waves' sums combine in wave order into the block's
// partial; blocks are summed in order by k_ghead_fin.
constexpr int kWC = 16;   // positions per wave chunk
constexpr size_t kWgLds = 64 * 1024;
static size_t ghead_lds_at(int tr, int W, int Cp) {
  return ((size_t)(tr + 2) * (W + 2) * 3 + 3) / 4 * 16 + (size_t)4 * kWC * (Cp + 4) * 4 + 3 * (size_t)Cp * 4 + 768 * 4;
}
// rows per weight-gradient block: about 2048 positions, fewer if the LDS tile would not fit
static int ghead_wrows(int W, int Cp) {
  int tr = std::max(1, std::min(16, 2048 / W));
  while (tr > 1 && ghead_lds_at(tr, W, Cp) > kWgLds) --tr;
  return tr;
}
static size_t ghead_wgrad_lds(int W, int Cp) { return ghead_lds_at(ghead_wrows(W, Cp), W, Cp); }

bool ghead_shape_ok(int W, int C) {
  const int Cp = (int)cpad(C);
  return C >= 1 && Cp <= 128 && W >= 4 && W % 4 == 0 && ghead_wgrad_lds(W, Cp) <= kWgLds;
}

template <int CT>   // CT = Cp / 32
__global__ __launch_bounds__(256, 2) void k_ghead_wgrad(const float* __restrict__ dimg, int ldd,
                                                        const float* __restrict__ img, const bf16_t* __restrict__ x,
                                                        int H, int W, FastDiv fdW, int C, int TRW,
                                                        const float* __restrict__ mean, const float* __restrict__ scale,
                                                        const float* __restrict__ shift, float* __restrict__ part) {
  constexpr int Cp = 32 * CT, AS = Cp + 4;
  extern __shared__ float4 sm4[];
  const int W2 = W + 2;
  float* const dts = reinterpret_cast<float*>(sm4);                  // [(rows + 2) * W2][3]
  float* const As = dts + ((TRW + 2) * W2 * 3 + 3) / 4 * 4;         // [4][kWC][AS]
  float4* const cst = reinterpret_cast<float4*>(As + 4 * kWC * AS);  // [3][Cp / 4]
  float* const sb = reinterpret_cast<float*>(cst + 3 * Cp / 4);      // [256][3] bias partials
  const int nrb = (H + TRW - 1) / TRW;
  const int b = blockIdx.x / nrb, h0 = (blockIdx.x % nrb) * TRW;
  const int nr = min(TRW, H - h0);
  const int tid = threadIdx.x, lane = tid & 63, kh = lane >> 5, ln = lane & 31;
  const int wv = tid >> 6;
  for (int c = tid; c < Cp; c += 256) {
    const bool ok = c < C;
    float* const cf = reinterpret_cast<float*>(cst);
    cf[c] = ok ? mean[c] : 0.f;
    cf[Cp + c] = ok ? scale[c] : 0.f;
    cf[2 * Cp + c] = ok ? shift[c] : 0.f;
  }
  float bs[3] = {0.f, 0.f, 0.f};
  for (int i = tid; i < (nr + 2) * W2; i += 256) {
    const int rr = i / W2, cc = i - rr * W2;
    const int h = h0 - 1 + rr, w = cc - 1;
    float d[3] = {0.f, 0.f, 0.f};
    if ((unsigned)h < (unsigned)H && (unsigned)w < (unsigned)W) {
      const int64_t q = ((int64_t)b * H + h) * W + w;
#pragma unroll
      for (int co = 0; co < 3; ++co) {
        const float y = img[q * 3 + co];
        d[co] = dimg[q * ldd + co] * (1.f - y * y);
      }
      if (rr >= 1 && rr <= nr) {
#pragma unroll
        for (int co = 0; co < 3; ++co) bs[co] += d[co];
      }
    }
#pragma unroll
    for (int co = 0; co < 3; ++co) dts[3 * i + co] = d[co];
  }
  // G column of this lane: dts offset relative to ((h - h0) * W2 + w) * 3
  const bool nok = ln < 27;
  const int co_n = ln / 9, tap = ln - 9 * co_n, tr = tap / 3, ts = tap - 3 * tr;
  const int boff = ((2 - tr) * W2 + (2 - ts)) * 3 + co_n;
  // staging role: position si of the chunk, channels 32 j + 8 sq + 0..7
  const int si = lane & 15, sq = lane >> 4;
  const int P = nr * W;
  const int nch = (P + kWC - 1) / kWC, iters = (nch + 3) / 4;
  uint4 xr[CT];
  // positions past P stage zeros (and meet a zero G row below)
  auto fetch = [&](int k) {
    const int p = k * kWC + si;
    const bool ok = k < nch && p < P;
    int64_t off = 0;
    if (ok) {
      const int h = (int)fdiv((uint32_t)p, fdW);
      off = (((int64_t)b * H + h0 + h) * W + (p - h * W)) * Cp + 8 * sq;
    }
#pragma unroll
    for (int j = 0; j < CT; ++j)
      xr[j] = ok ? *reinterpret_cast<const uint4*>(x + off + 32 * j) : make_uint4(0u, 0u, 0u, 0u);
  };
  f32x16 acc[CT];
#pragma unroll
  for (int ct = 0; ct < CT; ++ct)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[ct][r] = 0.f;
  fetch(wv);
  __syncthreads();
  float* const as = As + wv * kWC * AS;
  for (int it = 0; it < iters; ++it) {
    const int k = wv + 4 * it;
#pragma unroll
    for (int j = 0; j < CT; ++j) {
      const int q4 = 8 * j + 2 * sq;   // float4 index of channel 32 j + 8 sq
      float4 c[6];
#pragma unroll
      for (int a = 0; a < 3; ++a) {
        c[2 * a] = cst[a * (Cp / 4) + q4];
        c[2 * a + 1] = cst[a * (Cp / 4) + q4 + 1];
      }
      const float mu[8] = {c[0].x, c[0].y, c[0].z, c[0].w, c[1].x, c[1].y, c[1].z, c[1].w};
      const float sc[8] = {c[2].x, c[2].y, c[2].z, c[2].w, c[3].x, c[3].y, c[3].z, c[3].w};
      const float sh[8] = {c[4].x, c[4].y, c[4].z, c[4].w, c[5].x, c[5].y, c[5].z, c[5].w};
      float v[8], a[8];
      unpack8(xr[j], v);
#pragma unroll
      for (int e = 0; e < 8; ++e) a[e] = fmaxf((v[e] - mu[e]) * sc[e] + sh[e], 0.f);
      *reinterpret_cast<float4*>(as + si * AS + 32 * j + 8 * sq) = make_float4(a[0], a[1], a[2], a[3]);
      *reinterpret_cast<float4*>(as + si * AS + 32 * j + 8 * sq + 4) = make_float4(a[4], a[5], a[6], a[7]);
    }
    if (it + 1 < iters) fetch(k + 4);
    __syncthreads();
    if (k < nch) {
      // every operand of the chunk's k-steps first, then the products
      float av[kWC / 2][CT], bv[kWC / 2];
#pragma unroll
      for (int s = 0; s < kWC / 2; ++s) {
        const int pl = 2 * s + kh, p = k * kWC + pl;
        const int pc = min(p, P - 1);
        const int h = (int)fdiv((uint32_t)pc, fdW);
        const float g = dts[(h * W2 + (pc - h * W)) * 3 + boff];
        bv[s] = nok && p < P ? g : 0.f;
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) av[s][ct] = as[pl * AS + 32 * ct + ln];
      }
#pragma unroll
      for (int s = 0; s < kWC / 2; ++s)
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) acc[ct] = mfma_f32(av[s][ct], bv[s], acc[ct]);
    }
    __syncthreads();
  }
  // waves combine in order 0..3 (As is free after the loop's last barrier)
  float* const red = As;
  for (int w_ = 0; w_ < 4; ++w_) {
    if (wv == w_) {
#pragma unroll
      for (int ct = 0; ct < CT; ++ct)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int i = (ct * 16 + r) * 64 + lane;
          red[i] = w_ == 0 ? acc[ct][r] : red[i] + acc[ct][r];
        }
    }
    __syncthreads();
  }
  float* const out = part + (int64_t)blockIdx.x * (27 * C + 3);
  for (int i = tid; i < CT * 1024; i += 256) {
    const int l = i & 63, r = (i >> 6) & 15, ct = i >> 10;
    const int n = l & 31, c = 32 * ct + 8 * (r >> 2) + 4 * (l >> 5) + (r & 3);
    if (n < 27 && c < C) out[n * C + c] = red[i];
  }
  // bias: thread partials in thread order
#pragma unroll
  for (int co = 0; co < 3; ++co) sb[3 * tid + co] = bs[co];
  __syncthreads();
  if (tid < 3) {
    float v = 0.f;
    for (int j = 0; j < 256; ++j) v += sb[3 * j + tid];
    out[27 * C + tid] = v;
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

static int64_t ghead_wgrad_blocks(int B, int H, int W, int Cp) { return (int64_t)B * cdiv(H, ghead_wrows(W, Cp)); }

size_t ghead_ws_bytes(int B, int H, int W, int C) {
  return align256((size_t)ghead_wgrad_blocks(B, H, W, (int)cpad(C)) * (27 * C + 3) * 4);
}

void ghead_fwd(hipStream_t st, const void* x, int B, int H, int W, int C, int Cp, const float* mean,
               const float* scale, const float* shift, const float* Wt, const float* sigma, const float* bias,
               float* img) {
  const int TC = ghead_cols(W);
  const int64_t blocks = (int64_t)B * cdiv(H, kHR) * cdiv(W, TC);
  PG_CHECK(blocks < (1LL << 31) && Cp == cpad(C) && ghead_shape_ok(W, C), "ghead_fwd: shape");
  const bf16_t* xb = (const bf16_t*)x;
#define PG_GHF(CK)                                                                                              \
  hipLaunchKernelGGL(k_ghead_fwd<CK>, dim3((unsigned)blocks), dim3(256), 0, st, xb, H, W, C, TC, mean, scale, \
                     shift, Wt, sigma, bias, img)
  switch (Cp / 32) {
    case 1: PG_GHF(2); break;
    case 2: PG_GHF(4); break;
    case 3: PG_GHF(6); break;
    default: PG_GHF(8); break;
  }
#undef PG_GHF
  PG_LAUNCH_CHECK();
}

void ghead_bwd(hipStream_t st, const float* dimg, int ldd, const float* img, const void* x, int B, int H, int W,
               int C, int Cp, const float* mean, const float* scale, const float* shift, const float* Wt,
               const float* sigma, float* da, float* dwsn, float* dbias, void* ws) {
  const int64_t dblocks = (int64_t)B * cdiv(H, kDR) * cdiv(W, kDC);
  PG_CHECK(dblocks < (1LL << 31) && Cp == cpad(C) && ghead_shape_ok(W, C) && ldd >= 3, "ghead_bwd: shape");
  const int TRW = ghead_wrows(W, Cp);
  const size_t lds = ghead_wgrad_lds(W, Cp);
  const int nch = (int)ghead_wgrad_blocks(B, H, W, Cp);
  const FastDiv fdW = make_fastdiv((uint32_t)W);
  hipLaunchKernelGGL(k_ghead_dgrad, dim3((unsigned)dblocks), dim3(256), 27 * Cp * sizeof(float), st, dimg, ldd,
                     img, B, H, W, C, Cp, Wt, sigma, da);
  const bf16_t* xb = (const bf16_t*)x;
#define PG_GHW(CT)                                                                                                   \
  hipLaunchKernelGGL(k_ghead_wgrad<CT>, dim3(nch), dim3(256), lds, st, dimg, ldd, img, xb, H, W, fdW, C, TRW, mean,  \
                     scale, shift, (float*)ws)
  switch (Cp / 32) {
    case 1: PG_GHW(1); break;
    case 2: PG_GHW(2); break;
    case 3: PG_GHW(3); break;
    default: PG_GHW(4); break;
  }
#undef PG_GHW
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
  // relu(t) as (t > 0 ? t : 0) would drop a NaN logit; a NaN propagates
  // into the loss instead, so that a diverged discriminator is reported
  auto relu_nan = [](float t) { return t > 0.f || t != t ? t : 0.f; };
  for (int i = threadIdx.x; i < n; i += 256) {
    const float v = out[i];
    if (mode == 0) {
      if (i < nr) {
        s += (double)relu_nan(1.f - v) / nr;
        dout[i] = v < 1.f ? -1.f / nr : 0.f;
      } else {
        s += (double)relu_nan(1.f + v) / nf;
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

// --------------------------------------------------- optimisers
// Adam:      m = b1 m + (1-b1) g;  v = b2 v + (1-b2) g^2;  p -= lr_t m / (sqrt(v c2) + eps)
// AdaBelief: m = b1 m + (1-b1) g;  s = b2 s + (1-b2) (g - m)^2 + eps;
//            p -= lr_t m / (sqrt(s c2) + eps)
// with lr_t = lr / (1 - b1^t) and c2 = 1 / (1 - b2^t) (bias corrections).
// One element; four per thread through 16-byte accesses (28 bytes of HBM
// traffic per parameter either way).
template <int KIND>
PG_DEV void optim1(float& p, float g, float& m, float& v, float b1, float b2, float lr_t, float c2, float eps) {
  m = b1 * m + (1.f - b1) * g;
  if (KIND == 0) {
    v = b2 * v + (1.f - b2) * g * g;
  } else {
    const float d = g - m;
    v = b2 * v + (1.f - b2) * d * d + eps;
  }
  p -= lr_t * m / (sqrtf(v * c2) + eps);
}
template <int KIND>
__global__ void k_optim(float* p, const float* g, float* m, float* v, int64_t n, float b1, float b2, float lr_t,
                        float c2, float eps) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t n4 = n >> 2;
  if (i < n4) {
    float4 pp = reinterpret_cast<float4*>(p)[i], mm = reinterpret_cast<float4*>(m)[i];
    float4 vv = reinterpret_cast<float4*>(v)[i];
    const float4 gg = reinterpret_cast<const float4*>(g)[i];
    optim1<KIND>(pp.x, gg.x, mm.x, vv.x, b1, b2, lr_t, c2, eps);
    optim1<KIND>(pp.y, gg.y, mm.y, vv.y, b1, b2, lr_t, c2, eps);
    optim1<KIND>(pp.z, gg.z, mm.z, vv.z, b1, b2, lr_t, c2, eps);
    optim1<KIND>(pp.w, gg.w, mm.w, vv.w, b1, b2, lr_t, c2, eps);
    reinterpret_cast<float4*>(p)[i] = pp;
    reinterpret_cast<float4*>(m)[i] = mm;
    reinterpret_cast<float4*>(v)[i] = vv;
  } else if (i < n4 + (n & 3)) {
    const int64_t j = 4 * n4 + (i - n4);
    optim1<KIND>(p[j], g[j], m[j], v[j], b1, b2, lr_t, c2, eps);
  }
}

void optim_step(hipStream_t st, int kind, float* p, const float* g, float* m, float* v, int64_t n, float b1,
                float b2, float lr, float eps, int64_t t) {
  if (n <= 0) return;
  PG_CHECK((((uintptr_t)p | (uintptr_t)g | (uintptr_t)m | (uintptr_t)v) & 15) == 0,
           "optimiser: 16-byte aligned buffers");
  PG_CHECK(kind == 0 || kind == 1, "optimiser: unknown kind");
  const double lr_t = (double)lr / (1.0 - std::pow((double)b1, (double)t));
  const double c2 = 1.0 / (1.0 - std::pow((double)b2, (double)t));
  const int64_t threads = (n >> 2) + (n & 3);
  const dim3 grid((unsigned)cdiv(threads, 256));
  ProfScope ps(st);
  if (kind == 0)
    hipLaunchKernelGGL(k_optim<0>, grid, dim3(256), 0, st, p, g, m, v, n, b1, b2, (float)lr_t, (float)c2, eps);
  else
    hipLaunchKernelGGL(k_optim<1>, grid, dim3(256), 0, st, p, g, m, v, n, b1, b2, (float)lr_t, (float)c2, eps);
  // p, g, m, v read; p, m, v written
  ps.done_bytes(kind == 0 ? "k_optim<adam>" : "k_optim<adabelief>", 28.0 * n);
  PG_LAUNCH_CHECK();
}

}  // namespace pg
