// Implicit-GEMM convolutions for gfx950.
//
// Forward and data-gradient convolutions are one kernel: a GEMM with
// M = output pixels (NHWC rows), N = output channels, K = taps x input
// channels, where the A operand is gathered from the activation on the fly
// (im2col never exists in memory) and transformed while it is staged into
// LDS (BatchNorm affine, ReLU, nearest-upsample or sum-pool gather).  The
// data gradient is the same kernel run with spatially flipped, transposed
// weights.  The weight gradient is a GEMM over M (pixels) with both operands
// transposed in registers on the way into LDS, split over M with a
// fixed-order reduction (no float atomics: results are bitwise
// reproducible).
//
// bf16 path: v_mfma_f32_32x32x16_bf16, fp32 accumulation, 4 waves per
// 256-thread block, double-buffered LDS, one barrier per K step.
// fp32 path: a plain LDS-tiled SIMT GEMM (used by the fp32 block config and
// tests; the bf16 path is the performance path).
#include <cmath>

#include "ops.hpp"

namespace pg {

thread_local Profiler* t_prof = nullptr;

// ------------------------------------------------------------ A operand
struct AOp {
  const void* x;
  int B, Hx, Wx, C;
  float gscale;
  const float* mean;
  const float* scale;
  const float* shift;
  int tab_stride;
  int H, W, R, pad;
  int64_t M;
};

PG_DEV void decode_m(int64_t m, int H, int W, int quad, int& b, int& oh, int& ow) {
  if (!quad) {
    int64_t t = m / W;
    ow = (int)(m - t * W);
    b = (int)(t / H);
    oh = (int)(t - (int64_t)b * H);
  } else {
    const int W2 = W >> 1, H2 = H >> 1;
    const int qd = (int)(m & 3);
    const int64_t p = m >> 2;
    const int64_t t = p / W2;
    const int pw = (int)(p - t * W2);
    b = (int)(t / H2);
    const int ph = (int)(t - (int64_t)b * H2);
    oh = 2 * ph + (qd >> 1);
    ow = 2 * pw + (qd & 1);
  }
}

// Source element offsets of the gathered input at conv-grid position
// (ih, iw).  Returns the number of source pixels (1, or 4 for sum-pool).
template <int GATHER>
PG_DEV int src_offsets(const AOp& a, int b, int ih, int iw, int c, int64_t* off) {
  if (GATHER == G_DIRECT) {
    off[0] = (((int64_t)b * a.Hx + ih) * a.Wx + iw) * a.C + c;
    return 1;
  } else if (GATHER == G_UP2) {
    off[0] = (((int64_t)b * a.Hx + (ih >> 1)) * a.Wx + (iw >> 1)) * a.C + c;
    return 1;
  } else {
#pragma unroll
    for (int d = 0; d < 4; ++d)
      off[d] = (((int64_t)b * a.Hx + 2 * ih + (d >> 1)) * a.Wx + 2 * iw + (d & 1)) * a.C + c;
    return 4;
  }
}

// Apply gather-sum, scale, affine BN and ReLU to 8 consecutive channels.
template <int GATHER, bool AFF, bool RELU>
PG_DEV void xform8(const AOp& a, float* f, int b, int c) {
  const float gs = a.gscale;
#pragma unroll
  for (int i = 0; i < 8; ++i) f[i] *= gs;
  if (AFF) {
    const float4* mp = reinterpret_cast<const float4*>(a.mean + c);
    const float4* sp = reinterpret_cast<const float4*>(a.scale + (int64_t)b * a.tab_stride + c);
    const float4* hp = reinterpret_cast<const float4*>(a.shift + (int64_t)b * a.tab_stride + c);
    float4 m0 = mp[0], m1 = mp[1], s0 = sp[0], s1 = sp[1], h0 = hp[0], h1 = hp[1];
    const float mm[8] = {m0.x, m0.y, m0.z, m0.w, m1.x, m1.y, m1.z, m1.w};
    const float ss[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
    const float hh[8] = {h0.x, h0.y, h0.z, h0.w, h1.x, h1.y, h1.z, h1.w};
#pragma unroll
    for (int i = 0; i < 8; ++i) f[i] = (f[i] - mm[i]) * ss[i] + hh[i];
  }
  if (RELU) {
#pragma unroll
    for (int i = 0; i < 8; ++i) f[i] = fmaxf(f[i], 0.f);
  }
}

struct ConvK {
  AOp a;
  int cchunks, ksteps;
  const void* w;
  int Np;
  ConvOut o;
  int tiles_m, tiles_n;
};

PG_DEV int remap_tile(int bid, int total) {
  // Blocks are dispatched round-robin over the 8 XCDs; give each XCD a
  // contiguous run of tiles so neighbouring tiles share its L2.
  if ((total & 7) == 0) {
    const int per = total >> 3;
    return (bid & 7) * per + (bid >> 3);
  }
  return bid;
}

// Epilogue for one output element (non-pooled) or one pooled pixel.
PG_DEV void epi_store(const ConvK& k, int64_t mo, int col, float v, int H, int W) {
  const ConvOut& o = k.o;
  if (col >= o.n_real) {
    v = 0.f;
  } else {
    if (o.mask) {
      const int64_t mi = mo * o.maskC + col;
      const float mk = o.mask_f32 ? ((const float*)o.mask)[mi] : bf2f(((const bf16_t*)o.mask)[mi]);
      v = mk > 0.f ? v : 0.f;
    }
    if (o.res_mode != R_NONE) {
      int64_t ri;
      if (o.res_mode == R_SAME) {
        ri = mo * o.resC + col;
      } else {  // R_HALF: (h>>1, w>>1) of a half-resolution tensor
        int b, oh, ow;
        decode_m(mo, H, W, 0, b, oh, ow);
        ri = (((int64_t)b * (H >> 1) + (oh >> 1)) * (W >> 1) + (ow >> 1)) * o.resC + col;
      }
      const float rv = o.res_f32 ? ((const float*)o.res)[ri] : bf2f(((const bf16_t*)o.res)[ri]);
      v += o.res_scale * rv;
    }
  }
  if (o.y_f32)
    ((float*)o.y)[mo * o.yC + col] = v;
  else
    ((bf16_t*)o.y)[mo * o.yC + col] = f2bf(v);
}

// --------------------------------------------------------- bf16 MFMA conv
template <int WM, int WN, int TM, int TN, int GATHER, bool AFF, bool RELU>
__global__ __launch_bounds__(256, 2) void k_conv_mfma(ConvK k) {
  constexpr int BM = WM * TM * 32, BN = WN * TN * 32;
  constexpr int LDA = 40;                     // 32 bf16 + 8 pad per LDS row
  constexpr int AP = BM / 64;                 // A rows per thread
  constexpr int BP = (BN * 4 + 255) / 256;    // B 16-byte chunks per thread
  constexpr int NLD = GATHER == G_POOL2 ? 4 : 1;
  __shared__ __attribute__((aligned(16))) bf16_t As[2][BM * LDA];
  __shared__ __attribute__((aligned(16))) bf16_t Bs[2][BN * LDA];

  const AOp& a = k.a;
  const int bid = remap_tile(blockIdx.x, k.tiles_m * k.tiles_n);
  const int tmi = bid / k.tiles_n, tni = bid - tmi * k.tiles_n;
  const int64_t m0 = (int64_t)tmi * BM;
  const int n0 = tni * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int q = tid & 3;
  const int quad = k.o.pool;

  int rb[AP], roh[AP], row_[AP];
  bool rv[AP];
#pragma unroll
  for (int p = 0; p < AP; ++p) {
    const int64_t m = m0 + (tid >> 2) + 64 * p;
    rv[p] = m < a.M;
    decode_m(rv[p] ? m : 0, a.H, a.W, quad, rb[p], roh[p], row_[p]);
  }
  const bf16_t* X = (const bf16_t*)a.x;
  const bf16_t* Wt = (const bf16_t*)k.w;
  uint4 ra[AP][NLD];
  bool va[AP];
  uint4 rw[BP];
  const bool plain = !AFF && !RELU && GATHER != G_POOL2 && a.gscale == 1.f;
  const bool relu_only = !AFF && RELU && GATHER != G_POOL2 && a.gscale == 1.f;
  const int RR = a.R * a.R;

  auto load = [&](int ks) {
    const int tap = ks / k.cchunks;
    const int c0 = (ks - tap * k.cchunks) * 32;
    const int r = tap / a.R, s = tap - (tap / a.R) * a.R;
#pragma unroll
    for (int p = 0; p < AP; ++p) {
      const int ih = roh[p] + r - a.pad, iw = row_[p] + s - a.pad;
      const bool v = rv[p] && ih >= 0 && ih < a.H && iw >= 0 && iw < a.W;
      va[p] = v;
      if (v) {
        int64_t off[4];
        src_offsets<GATHER>(a, rb[p], ih, iw, c0 + q * 8, off);
#pragma unroll
        for (int d = 0; d < NLD; ++d) ra[p][d] = *reinterpret_cast<const uint4*>(X + off[d]);
      }
    }
#pragma unroll
    for (int p = 0; p < BP; ++p) {
      const int idx = tid + 256 * p;
      const int n = n0 + (idx >> 2);
      if (idx < BN * 4 && n < k.Np)
        rw[p] = *reinterpret_cast<const uint4*>(Wt + ((int64_t)n * RR + tap) * a.C + c0 + (idx & 3) * 8);
      else
        rw[p] = make_uint4(0, 0, 0, 0);
    }
  };
  auto store = [&](int ks, int buf) {
    const int tap = ks / k.cchunks;
    const int c0 = (ks - tap * k.cchunks) * 32;
#pragma unroll
    for (int p = 0; p < AP; ++p) {
      uint4 out = make_uint4(0, 0, 0, 0);
      if (va[p]) {
        if (plain) {
          out = ra[p][0];
        } else if (relu_only) {
          out = relu8_bits(ra[p][0]);
        } else {
          float f[8];
          unpack8(ra[p][0], f);
#pragma unroll
          for (int d = 1; d < NLD; ++d) {
            float g[8];
            unpack8(ra[p][d], g);
#pragma unroll
            for (int i = 0; i < 8; ++i) f[i] += g[i];
          }
          xform8<GATHER, AFF, RELU>(a, f, rb[p], c0 + q * 8);
          out = pack8(f);
        }
      }
      *reinterpret_cast<uint4*>(&As[buf][((tid >> 2) + 64 * p) * LDA + q * 8]) = out;
    }
#pragma unroll
    for (int p = 0; p < BP; ++p) {
      const int idx = tid + 256 * p;
      if (idx < BN * 4) *reinterpret_cast<uint4*>(&Bs[buf][(idx >> 2) * LDA + (idx & 3) * 8]) = rw[p];
    }
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  load(0);
  store(0, 0);
  __syncthreads();
  int buf = 0;
  for (int ks = 0; ks < k.ksteps; ++ks) {
    const bool more = ks + 1 < k.ksteps;
    if (more) load(ks + 1);
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      bf16x8 av[TM], bv[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        av[i] = *reinterpret_cast<const bf16x8*>(
            &As[buf][((wm * TM + i) * 32 + (lane & 31)) * LDA + kk * 16 + (lane >> 5) * 8]);
#pragma unroll
      for (int j = 0; j < TN; ++j)
        bv[j] = *reinterpret_cast<const bf16x8*>(
            &Bs[buf][((wn * TN + j) * 32 + (lane & 31)) * LDA + kk * 16 + (lane >> 5) * 8]);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[i], bv[j], acc[i][j], 0, 0, 0);
    }
    if (more) store(ks + 1, buf ^ 1);
    __syncthreads();
    buf ^= 1;
  }

  // epilogue
  const float accs = (k.o.acc_scale ? *k.o.acc_scale : 1.f) * k.o.acc_mul / (k.o.acc_div ? *k.o.acc_div : 1.f);
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int col = n0 + (wn * TN + j) * 32 + (lane & 31);
      if (col >= k.o.yC) continue;
      const float bias = (k.o.bias && col < k.o.n_real) ? k.o.bias[col] : 0.f;
      const int64_t rbase = m0 + (wm * TM + i) * 32 + 4 * (lane >> 5);
      if (!k.o.pool) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int64_t m = rbase + 8 * (r >> 2) + (r & 3);
          if (m < a.M) epi_store(k, m, col, acc[i][j][r] * accs + bias, a.H, a.W);
        }
      } else {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int64_t m = rbase + 8 * g;
          if (m < a.M) {
            const float v = 0.25f * ((acc[i][j][4 * g] + acc[i][j][4 * g + 1]) +
                                     (acc[i][j][4 * g + 2] + acc[i][j][4 * g + 3]));
            epi_store(k, m >> 2, col, v * accs + bias, a.H, a.W);
          }
        }
      }
    }
  }
}

// ------------------------------------------------------ fp32 MFMA conv
// The fp32 path (exact-fp32 configurations) on the fp32 matrix cores:
// 64 x 64 tiles (pixels x output channels), 16-deep K steps staged in LDS
// k-major, four waves each owning a 32 x 32 quarter through
// v_mfma_f32_32x32x2_f32 (a lane supplies one value of each operand per
// instruction: row lane % 32 at K index lane / 32).  Weights are the A
// operand (rows = output channels), pixels the B operand, so a lane ends
// with one pixel (lane % 32) and the 16 channels (r % 4) + 8 (r / 4) +
// 4 (lane / 32) of its wave's 32.
template <int GATHER, bool AFF, bool RELU>
__global__ __launch_bounds__(256) void k_conv_f32mfma(ConvK k) {
  __shared__ float As[16][68];
  __shared__ float Bs[16][68];
  const AOp& a = k.a;
  const int bid = blockIdx.x;
  const int tmi = bid / k.tiles_n, tni = bid - tmi * k.tiles_n;
  const int64_t m0 = (int64_t)tmi * 64;
  const int n0 = tni * 64;
  const int tid = threadIdx.x, lane = tid & 63, l32 = lane & 31, kh = lane >> 5;
  const int wave = tid >> 6, wm = wave >> 1, wn = wave & 1;
  const int arow = tid >> 2, c4 = (tid & 3) * 4;
  const int64_t am = m0 + arow;
  const bool arv = am < a.M;
  int b, oh, ow;
  decode_m(arv ? am : 0, a.H, a.W, k.o.pool, b, oh, ow);
  const float* X = (const float*)a.x;
  const float* Wt = (const float*)k.w;
  const int RR = a.R * a.R;
  f32x16 acc;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[r] = 0.f;
  for (int ks = 0; ks < k.ksteps; ++ks) {
    const int tap = ks / k.cchunks;
    const int c0 = (ks - tap * k.cchunks) * 16;
    const int r = tap / a.R, s = tap - (tap / a.R) * a.R;
    const int ih = oh + r - a.pad, iw = ow + s - a.pad;
    float f[4] = {0.f, 0.f, 0.f, 0.f};
    if (arv && ih >= 0 && ih < a.H && iw >= 0 && iw < a.W) {
      int64_t off[4];
      const int n = src_offsets<GATHER>(a, b, ih, iw, c0 + c4, off);
      for (int d = 0; d < n; ++d) {
        const float4 v = *reinterpret_cast<const float4*>(X + off[d]);
        f[0] += v.x; f[1] += v.y; f[2] += v.z; f[3] += v.w;
      }
      const int c = c0 + c4;
      for (int i = 0; i < 4; ++i) {
        float t = f[i] * a.gscale;
        if (AFF) t = (t - a.mean[c + i]) * a.scale[(int64_t)b * a.tab_stride + c + i] +
                     a.shift[(int64_t)b * a.tab_stride + c + i];
        if (RELU) t = fmaxf(t, 0.f);
        f[i] = t;
      }
    }
    for (int i = 0; i < 4; ++i) As[c4 + i][arow] = f[i];
    const int n = n0 + arow;
    float4 wv = make_float4(0.f, 0.f, 0.f, 0.f);
    if (n < k.Np) wv = *reinterpret_cast<const float4*>(Wt + ((int64_t)n * RR + tap) * a.C + c0 + c4);
    Bs[c4 + 0][arow] = wv.x; Bs[c4 + 1][arow] = wv.y; Bs[c4 + 2][arow] = wv.z; Bs[c4 + 3][arow] = wv.w;
    __syncthreads();
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const float wa = Bs[2 * t + kh][wn * 32 + l32];
      const float xb = As[2 * t + kh][wm * 32 + l32];
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(wa, xb, acc, 0, 0, 0);
    }
    __syncthreads();
  }
  const float accs = (k.o.acc_scale ? *k.o.acc_scale : 1.f) * k.o.acc_mul / (k.o.acc_div ? *k.o.acc_div : 1.f);
  const int64_t m = m0 + wm * 32 + l32;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int col = n0 + wn * 32 + (r & 3) + 8 * (r >> 2) + 4 * kh;
    const float bias = (k.o.bias && col < k.o.n_real) ? k.o.bias[col] : 0.f;
    if (!k.o.pool) {
      if (col < k.o.yC && m < a.M) epi_store(k, m, col, acc[r] * accs + bias, a.H, a.W);
    } else {
      // pooled output: the 2 x 2 window is four consecutive rows m (tiles
      // hold whole windows), here four consecutive lanes, summed in the
      // order (m0 + m1) + (m2 + m3)
      float v = acc[r];
      v += __shfl_xor(v, 1);
      v += __shfl_xor(v, 2);
      if ((lane & 3) == 0 && col < k.o.yC && m < a.M) epi_store(k, m >> 2, col, 0.25f * v * accs + bias, a.H, a.W);
    }
  }
}

// --------------------------------------------------------------- launcher
static std::string kname(const char* base, std::initializer_list<int> args);

static std::string kname(const char* base, std::initializer_list<int> args) {
  std::string n = std::string(base) + "<";
  bool first = true;
  for (int a : args) {
    n += (first ? "" : ",") + std::to_string(a);
    first = false;
  }
  return n + ">";
}

// returns the launched kernel's name (template instance)
template <int WM, int WN, int TM, int TN>
static std::string launch_mfma_cfg(hipStream_t s, ConvK& k, int gather, bool aff, bool relu) {
  constexpr int BM = WM * TM * 32, BN = WN * TN * 32;
  k.tiles_m = (int)cdiv(k.a.M, BM);
  k.tiles_n = (int)cdiv(k.Np, BN);
  dim3 grid(k.tiles_m * k.tiles_n), block(256);
#define PG_CONV_CASE(G, A_, R_)                                                   \
  if (gather == G && aff == A_ && relu == R_) {                                   \
    hipLaunchKernelGGL((k_conv_mfma<WM, WN, TM, TN, G, A_, R_>), grid, block, 0, s, k); \
    return kname("k_conv_mfma", {WM, WN, TM, TN, G, A_, R_});                   \
  }
  PG_CONV_CASE(G_DIRECT, false, false)
  PG_CONV_CASE(G_DIRECT, false, true)
  PG_CONV_CASE(G_DIRECT, true, true)
  PG_CONV_CASE(G_UP2, false, false)
  PG_CONV_CASE(G_UP2, true, true)
  PG_CONV_CASE(G_POOL2, false, false)
#undef PG_CONV_CASE
  throw Error{-2, "conv: unsupported prologue combination"};
}

void conv_fwd(hipStream_t s, bool f32, const ConvIn& in, int H, int W, int R,
              const void* w, int Np, const ConvOut& out) {
  ConvK k;
  k.a = AOp{in.x, in.B, in.Hx, in.Wx, in.C, in.gscale, in.mean, in.scale, in.shift,
            in.tab_stride, H, W, R, R / 2, (int64_t)in.B * H * W};
  k.w = w;
  k.Np = Np;
  k.o = out;
  if (k.a.M == 0) return;
  const bool aff = in.mean != nullptr;
  ProfScope prof(s);
  // (the sub-pixel gather runs four parity classes over the M source pixels)
  const double flops = 2.0 * (double)k.a.M * out.n_real * R * R * (in.c_real ? in.c_real : in.C) *
                       (in.gather == G_SUB ? 4 : 1);
  if (f32) {
    k.cchunks = in.C / 16;
    k.ksteps = R * R * k.cchunks;
    k.tiles_m = (int)cdiv(k.a.M, 64);
    k.tiles_n = (int)cdiv(Np, 64);
    dim3 grid(k.tiles_m * k.tiles_n), block(256);
#define PG_F32_CASE(G, A_, R_)                                                     \
  if (in.gather == G && aff == A_ && (bool)in.relu == R_) {                         \
    hipLaunchKernelGGL((k_conv_f32mfma<G, A_, R_>), grid, block, 0, s, k);             \
    PG_LAUNCH_CHECK();                                                              \
    prof.done(kname("k_conv_f32mfma", {G, A_, R_}), flops);                            \
    return;                                                                         \
  }
    PG_F32_CASE(G_DIRECT, false, false)
    PG_F32_CASE(G_DIRECT, false, true)
    PG_F32_CASE(G_DIRECT, true, true)
    PG_F32_CASE(G_UP2, false, false)
    PG_F32_CASE(G_UP2, true, true)
    PG_F32_CASE(G_POOL2, false, false)
#undef PG_F32_CASE
    throw Error{-2, "conv(f32): unsupported prologue combination"};
  }
  k.cchunks = in.C / 32;
  k.ksteps = R * R * k.cchunks;
  // A positive power-of-two operand scale is exact in bf16 and fp32: move it
  // to the epilogue so the streamlined kernel applies.
  if (!aff && in.gather != G_POOL2 && k.a.gscale > 0.f && k.a.gscale != 1.f) {
    int e2;
    if (std::frexp(k.a.gscale, &e2) == 0.5f) {
      k.o.acc_mul *= k.a.gscale;
      k.a.gscale = 1.f;
    }
  }
  {
    ConvIn in2 = in;
    in2.gscale = k.a.gscale;
    if (conv_fwd_mfma_ok(in2, H, W, R, Np, k.o)) {
      const std::string name = conv_fwd_mfma(s, in2, H, W, R, w, Np, k.o);
      PG_LAUNCH_CHECK();
      prof.done(name, flops, k.a.M, Np, (int64_t)R * R * in.C);
      return;
    }
  }
  // tile choice: 128x128 when N is a multiple of 128, else 256x96 / 128x64
  // shapes so that BigGAN's 96-multiple widths waste no MMA columns.
  std::string name;
  if (Np % 128 == 0)
    name = launch_mfma_cfg<2, 2, 2, 2>(s, k, in.gather, aff, in.relu);
  else if (Np % 96 == 0)
    name = launch_mfma_cfg<4, 1, 2, 3>(s, k, in.gather, aff, in.relu);
  else if (Np <= 64)
    name = launch_mfma_cfg<4, 1, 1, 2>(s, k, in.gather, aff, in.relu);
  else
    name = launch_mfma_cfg<2, 2, 2, 2>(s, k, in.gather, aff, in.relu);
  PG_LAUNCH_CHECK();
  prof.done(name, flops, k.a.M, Np, (int64_t)R * R * in.C);
}

// ================================================================ wgrad
struct WgK {
  AOp a;
  const void* g;
  int gHs, gWs, gC, g_gather;
  int Np, Kdim;
  int64_t m_per_split;
  int splits, tiles_n, tiles_k;
  float* part;   // [splits][Np][Kdim]
};

PG_DEV uint32_t word_of(const uint4& v, int i) {
  return i == 0 ? v.x : (i == 1 ? v.y : (i == 2 ? v.z : v.w));
}

// 8x8 transpose of bf16: in[i] holds row i (8 values), out[j] holds column j.
PG_DEV void transpose8(const uint4* in, uint4* out) {
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    uint32_t w[4];
    const uint32_t sel = (j & 1) ? 0x07060302u : 0x05040100u;
#pragma unroll
    for (int t = 0; t < 4; ++t)
      w[t] = __builtin_amdgcn_perm(word_of(in[2 * t + 1], j >> 1), word_of(in[2 * t], j >> 1), sel);
    out[j] = make_uint4(w[0], w[1], w[2], w[3]);
  }
}

// advance (b, oh, ow) by one pixel in NHWC order
PG_DEV void step_pix(int& b, int& oh, int& ow, int H, int W) {
  if (++ow == W) {
    ow = 0;
    if (++oh == H) { oh = 0; ++b; }
  }
}

template <int GATHER, bool AFF, bool RELU>
__global__ __launch_bounds__(256, 2) void k_wgrad_mfma(WgK k) {
  constexpr int LDT = 72;    // 64 m + 8 pad (bf16) per LDS row
  __shared__ __attribute__((aligned(16))) bf16_t Gt[2][128 * LDT];
  __shared__ __attribute__((aligned(16))) bf16_t Xt[2][128 * LDT];
  const AOp& a = k.a;
  const int tiles = k.tiles_n * k.tiles_k;
  const int split = blockIdx.x / tiles;
  const int tile = blockIdx.x - split * tiles;
  const int tni = tile / k.tiles_k, tki = tile - tni * k.tiles_k;
  const int n0 = tni * 128, k0 = tki * 128;
  const int64_t mbeg = (int64_t)split * k.m_per_split;
  int64_t mend = mbeg + k.m_per_split;
  if (mend > a.M) mend = a.M;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  // loader role: threads 0..127 load the gradient, 128..255 the im2col
  const bool isg = tid < 128;
  const int sb = tid & 127;
  const int mg = sb >> 4, cg = sb & 15;     // 8 m-groups x 16 column groups
  const int col = (isg ? n0 : k0) + cg * 8;
  // im2col column -> (tap, channel)
  const int tap = col / a.C, cch = col - (col / a.C) * a.C;
  const int tr = tap / a.R, tsx = tap - (tap / a.R) * a.R;
  const bool colv = isg ? (col < k.Np) : (col < k.Kdim);
  const bf16_t* G = (const bf16_t*)k.g;
  const bf16_t* X = (const bf16_t*)a.x;
  const bool plainx = !AFF && !RELU && GATHER != G_POOL2 && a.gscale == 1.f;
  const bool reluonly = !AFF && RELU && GATHER != G_POOL2 && a.gscale == 1.f;
  constexpr int NLD = GATHER == G_POOL2 ? 4 : 1;

  uint4 raw[8][NLD];
  bool rvld[8];
  int rbb[8];

  auto load = [&](int64_t mc) {
    const int64_t mrow = mc + mg * 8;
    int b = 0, oh = 0, ow = 0;
    if (mrow < mend) decode_m(mrow, a.H, a.W, 0, b, oh, ow);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const bool inm = mrow + i < mend;
      rbb[i] = b;
      bool v = false;
      if (isg) {
        v = inm && colv;
        if (v) {
          int64_t off;
          if (k.g_gather == G_DIRECT)
            off = (mrow + i) * k.gC + col;
          else
            off = (((int64_t)b * k.gHs + (oh >> 1)) * k.gWs + (ow >> 1)) * k.gC + col;
          raw[i][0] = *reinterpret_cast<const uint4*>(G + off);
        }
      } else {
        const int ih = oh + tr - a.pad, iw = ow + tsx - a.pad;
        v = inm && colv && ih >= 0 && ih < a.H && iw >= 0 && iw < a.W;
        if (v) {
          int64_t off[4];
          src_offsets<GATHER>(a, b, ih, iw, cch, off);
#pragma unroll
          for (int d = 0; d < NLD; ++d) raw[i][d] = *reinterpret_cast<const uint4*>(X + off[d]);
        }
      }
      rvld[i] = v;
      if (inm) step_pix(b, oh, ow, a.H, a.W);
    }
  };
  auto store = [&](int buf) {
    uint4 rows[8], cols[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      rows[i] = make_uint4(0, 0, 0, 0);
      if (rvld[i]) {
        if (isg || plainx) {
          rows[i] = raw[i][0];
        } else if (reluonly) {
          rows[i] = relu8_bits(raw[i][0]);
        } else {
          float f[8];
          unpack8(raw[i][0], f);
#pragma unroll
          for (int d = 1; d < NLD; ++d) {
            float g2[8];
            unpack8(raw[i][d], g2);
#pragma unroll
            for (int e = 0; e < 8; ++e) f[e] += g2[e];
          }
          xform8<GATHER, AFF, RELU>(a, f, rbb[i], cch);
          rows[i] = pack8(f);
        }
      }
    }
    transpose8(rows, cols);
    bf16_t* dst = isg ? Gt[buf] : Xt[buf];
#pragma unroll
    for (int j = 0; j < 8; ++j)
      *reinterpret_cast<uint4*>(&dst[(cg * 8 + j) * LDT + mg * 8]) = cols[j];
  };

  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int nsteps = (int)cdiv(mend - mbeg, 64);
  if (nsteps > 0) {
    load(mbeg);
    store(0);
  }
  __syncthreads();
  int buf = 0;
  for (int st = 0; st < nsteps; ++st) {
    const bool more = st + 1 < nsteps;
    if (more) load(mbeg + (int64_t)(st + 1) * 64);
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      bf16x8 av[2], bv[2];
#pragma unroll
      for (int i = 0; i < 2; ++i)
        av[i] = *reinterpret_cast<const bf16x8*>(
            &Gt[buf][((wm * 2 + i) * 32 + (lane & 31)) * LDT + kk * 16 + (lane >> 5) * 8]);
#pragma unroll
      for (int j = 0; j < 2; ++j)
        bv[j] = *reinterpret_cast<const bf16x8*>(
            &Xt[buf][((wn * 2 + j) * 32 + (lane & 31)) * LDT + kk * 16 + (lane >> 5) * 8]);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[i], bv[j], acc[i][j], 0, 0, 0);
    }
    if (more) store(buf ^ 1);
    __syncthreads();
    buf ^= 1;
  }
  float* part = k.part + (int64_t)split * k.Np * k.Kdim;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int kc = k0 + (wn * 2 + j) * 32 + (lane & 31);
      if (kc >= k.Kdim) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int n = n0 + (wm * 2 + i) * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        if (n < k.Np) part[(int64_t)n * k.Kdim + kc] = acc[i][j][r];
      }
    }
}

// fp32 weight gradient on the fp32 matrix cores: 64 (n) x 64 (k) tile, 16
// pixels per step staged in LDS, four waves each owning a 32 x 32 quarter
// through v_mfma_f32_32x32x2_f32 (the gradient is the A operand, rows =
// output channels; the gathered activation the B operand, columns = K).
template <int GATHER, bool AFF, bool RELU>
__global__ __launch_bounds__(256) void k_wgrad_f32mfma(WgK k) {
  __shared__ float Gs[16][68];
  __shared__ float Xs[16][68];
  const AOp& a = k.a;
  const int tiles = k.tiles_n * k.tiles_k;
  const int split = blockIdx.x / tiles;
  const int tile = blockIdx.x - split * tiles;
  const int tni = tile / k.tiles_k, tki = tile - tni * k.tiles_k;
  const int n0 = tni * 64, k0 = tki * 64;
  const int64_t mbeg = (int64_t)split * k.m_per_split;
  int64_t mend = mbeg + k.m_per_split;
  if (mend > a.M) mend = a.M;
  const int tid = threadIdx.x, lane = tid & 63, l32 = lane & 31, kh = lane >> 5;
  const int wave = tid >> 6, wn = wave >> 1, wk = wave & 1;
  const int lrow = tid >> 4, lc4 = (tid & 15) * 4;   // 16 pixels x 64 columns
  const float* G = (const float*)k.g;
  const float* X = (const float*)a.x;
  f32x16 acc;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[r] = 0.f;
  for (int64_t mc = mbeg; mc < mend; mc += 16) {
    const int64_t m = mc + lrow;
    float gv[4] = {0.f, 0.f, 0.f, 0.f}, xv[4] = {0.f, 0.f, 0.f, 0.f};
    if (m < mend) {
      int b, oh, ow;
      decode_m(m, a.H, a.W, 0, b, oh, ow);
      const int n = n0 + lc4;
      if (n < k.Np) {
        int64_t off = k.g_gather == G_DIRECT
                          ? m * k.gC + n
                          : (((int64_t)b * k.gHs + (oh >> 1)) * k.gWs + (ow >> 1)) * k.gC + n;
        const float4 v = *reinterpret_cast<const float4*>(G + off);
        gv[0] = v.x; gv[1] = v.y; gv[2] = v.z; gv[3] = v.w;
      }
      const int kc = k0 + lc4;
      if (kc < k.Kdim) {
        const int tap = kc / a.C, c = kc - (kc / a.C) * a.C;
        const int r = tap / a.R, s = tap - (tap / a.R) * a.R;
        const int ih = oh + r - a.pad, iw = ow + s - a.pad;
        if (ih >= 0 && ih < a.H && iw >= 0 && iw < a.W) {
          int64_t off[4];
          const int nl = src_offsets<GATHER>(a, b, ih, iw, c, off);
          for (int d = 0; d < nl; ++d) {
            const float4 v = *reinterpret_cast<const float4*>(X + off[d]);
            xv[0] += v.x; xv[1] += v.y; xv[2] += v.z; xv[3] += v.w;
          }
          for (int i = 0; i < 4; ++i) {
            float t = xv[i] * a.gscale;
            if (AFF) t = (t - a.mean[c + i]) * a.scale[(int64_t)b * a.tab_stride + c + i] +
                         a.shift[(int64_t)b * a.tab_stride + c + i];
            if (RELU) t = fmaxf(t, 0.f);
            xv[i] = t;
          }
        }
      }
    }
    for (int i = 0; i < 4; ++i) { Gs[lrow][lc4 + i] = gv[i]; Xs[lrow][lc4 + i] = xv[i]; }
    __syncthreads();
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const float ga = Gs[2 * t + kh][wn * 32 + l32];
      const float xb = Xs[2 * t + kh][wk * 32 + l32];
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(ga, xb, acc, 0, 0, 0);
    }
    __syncthreads();
  }
  float* part = k.part + (int64_t)split * k.Np * k.Kdim;
  const int kc = k0 + wk * 32 + l32;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int n = n0 + wn * 32 + (r & 3) + 8 * (r >> 2) + 4 * kh;
    if (n < k.Np && kc < k.Kdim) part[(int64_t)n * k.Kdim + kc] = acc[r];
  }
}

// dw = scale * sum over splits, in split order.
__global__ void k_split_reduce(const float* part, int splits, int64_t n, float scale, float* out) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  float s = 0.f;
  for (int j = 0; j < splits; ++j) s += part[(int64_t)j * n + i];
  out[i] = s * scale;
}

static void wgrad_plan(bool f32, int64_t M, int R, int Cin, int Np, int n_cu,
                       int& tiles_n, int& tiles_k, int& splits, int64_t& mps) {
  const int T = f32 ? 64 : 128;
  const int64_t Kdim = (int64_t)R * R * Cin;
  tiles_n = (int)cdiv(Np, T);
  tiles_k = (int)cdiv(Kdim, T);
  const int64_t tiles = (int64_t)tiles_n * tiles_k;
  const int64_t want = 4LL * n_cu;             // ~2 waves of 2 blocks per CU
  int64_t sp = cdiv(want, tiles);
  const int64_t minrows = f32 ? 256 : 1024;    // keep each split's K-loop long
  sp = std::min<int64_t>(sp, std::max<int64_t>(1, M / minrows));
  // cap the partial buffer at 512 MB
  const int64_t cap = (512LL << 20) / (4 * (int64_t)Np * Kdim);
  sp = std::max<int64_t>(1, std::min<int64_t>(sp, cap));
  const int64_t step = f32 ? 16 : 64;
  mps = cdiv(cdiv(M, sp), step) * step;
  splits = (int)cdiv(M, mps);
  if (splits < 1) splits = 1;
}

size_t conv_wgrad_ws(bool f32, int64_t M, int R, int Cin, int Np, int n_cu) {
  int tn, tk, sp;
  int64_t mps;
  wgrad_plan(f32, M, R, Cin, Np, n_cu, tn, tk, sp, mps);
  const size_t legacy = sp > 1 ? align256((size_t)sp * Np * R * R * Cin * 4) : 0;
  return f32 ? legacy : std::max(legacy, wgrad_tr_ws(M, R, Cin, Np, n_cu));
}

void conv_wgrad(hipStream_t s, bool f32, const GradIn& g, const ConvIn& in, int H, int W,
                int R, int Np, float* dw, void* ws, size_t ws_bytes, int n_cu) {
  const double flops =
      2.0 * (double)in.B * H * W * (g.n_real ? g.n_real : Np) * R * R * (in.c_real ? in.c_real : in.C);
  if (!f32 && wgrad_tr_ok(g, in, H, W, R, Np)) {
    if ((int64_t)in.B * H * W > 0) wgrad_tr(s, g, in, H, W, R, Np, dw, ws, ws_bytes, n_cu, flops);
    return;
  }
  WgK k;
  k.a = AOp{in.x, in.B, in.Hx, in.Wx, in.C, in.gscale, in.mean, in.scale, in.shift,
            in.tab_stride, H, W, R, R / 2, (int64_t)in.B * H * W};
  k.g = g.g;
  k.gHs = g.Hs;
  k.gWs = g.Ws;
  k.gC = g.C;
  k.g_gather = g.gather;
  k.Np = Np;
  k.Kdim = R * R * in.C;
  wgrad_plan(f32, k.a.M, R, in.C, Np, n_cu, k.tiles_n, k.tiles_k, k.splits, k.m_per_split);
  const int64_t nout = (int64_t)Np * k.Kdim;
  const bool direct = k.splits == 1 && g.gscale == 1.f;
  if (!direct && k.splits > 1 && (size_t)k.splits * nout * 4 > ws_bytes)
    throw Error{-3, "conv_wgrad: workspace too small"};
  k.part = direct || k.splits == 1 ? dw : (float*)ws;
  const bool aff = in.mean != nullptr;
  dim3 grid(k.splits * k.tiles_n * k.tiles_k), block(256);
  bool done = false;
  ProfScope prof(s);
  std::string name;
#define PG_WG_CASE(G, A_, R_)                                                   \
  if (!done && in.gather == G && aff == A_ && (bool)in.relu == R_) {            \
    if (f32)                                                                    \
      hipLaunchKernelGGL((k_wgrad_f32mfma<G, A_, R_>), grid, block, 0, s, k);      \
    else                                                                        \
      hipLaunchKernelGGL((k_wgrad_mfma<G, A_, R_>), grid, block, 0, s, k);      \
    name = kname(f32 ? "k_wgrad_f32mfma" : "k_wgrad_mfma", {G, A_, R_});            \
    done = true;                                                                \
  }
  PG_WG_CASE(G_DIRECT, false, false)
  PG_WG_CASE(G_DIRECT, false, true)
  PG_WG_CASE(G_DIRECT, true, true)
  PG_WG_CASE(G_UP2, false, false)
  PG_WG_CASE(G_UP2, true, true)
  PG_WG_CASE(G_POOL2, false, false)
#undef PG_WG_CASE
  if (!done) throw Error{-2, "conv_wgrad: unsupported prologue combination"};
  PG_LAUNCH_CHECK();
  prof.done(name, flops, k.a.M, Np, k.Kdim);
  if (k.splits > 1 || g.gscale != 1.f) {
    hipLaunchKernelGGL(k_split_reduce, dim3((unsigned)cdiv(nout, 256)), dim3(256), 0, s,
                       k.part, k.splits, nout, g.gscale, dw);
    PG_LAUNCH_CHECK();
  }
}

}  // namespace pg
