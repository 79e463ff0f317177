// Implicit-GEMM convolution (forward and data gradient) on gfx950 MFMA for
// the direct and nearest-upsample gathers with a plain or ReLU'd operand.
//
// GEMM: rows = output channels n (the packed weights, K contiguous), columns
// = output pixels m (the im2col of the activation, gathered on the fly), K =
// taps x input channels.  With the weights as the MFMA A operand each lane's
// accumulator holds four consecutive output channels of one pixel, so the
// epilogue (bias, ReLU mask, residual, 2x2 average pool, scale) works on
// 4-channel vectors and stores 8 bytes (bf16) or 16 bytes (fp32) per lane.
//
// K loop: tap-outer, channel-inner; a thread's source offsets are computed
// once per tap and advance by 32 channels per step.  Double-buffered LDS
// with one barrier per step; 64-byte LDS rows (32 bf16 of K) with the
// 16-byte chunks XOR-swizzled by row so that both the staging stores and
// the MFMA operand reads are free of bank conflicts.
#include "ops.hpp"

namespace pg {

namespace {

struct CfK {
  const bf16_t* x;
  const bf16_t* w;
  int64_t x_bytes, w_bytes;
  int Hx, Wx, C;        // activation source (C = channel stride)
  int H, W, R, pad;     // conv grid
  int M, Np, ksteps;
  FastDiv fdW, fdH, fdW2, fdH2;
  int tiles_m, tiles_n;
  ConvOut o;
};

PG_DEV int remap_tile2(int bid, int total) {
  // Blocks are dispatched round-robin over the 8 XCDs; give each XCD a
  // contiguous run of tiles so neighbouring tiles share its L2.
  if ((total & 7) == 0) {
    const int per = total >> 3;
    return (bid & 7) * per + (bid >> 3);
  }
  return bid;
}

// conv-grid position of output row m (quad-ordered rows list the four
// pixels of each 2x2 pooling window consecutively)
PG_DEV void pix_of(const CfK& k, int m, bool quad, int& b, int& oh, int& ow) {
  if (!quad) {
    const int t = (int)fdiv((uint32_t)m, k.fdW);
    ow = m - t * k.W;
    b = (int)fdiv((uint32_t)t, k.fdH);
    oh = t - b * k.H;
  } else {
    const int qd = m & 3, p = m >> 2;
    const int t = (int)fdiv((uint32_t)p, k.fdW2);
    const int pw = p - t * (k.W >> 1);
    b = (int)fdiv((uint32_t)t, k.fdH2);
    const int ph = t - b * (k.H >> 1);
    oh = 2 * ph + (qd >> 1);
    ow = 2 * pw + (qd & 1);
  }
}

PG_DEV void load4(const void* p, bool f32, int i, float* v) {
  if (f32) {
    const float4 q = *reinterpret_cast<const float4*>((const float*)p + i);
    v[0] = q.x; v[1] = q.y; v[2] = q.z; v[3] = q.w;
  } else {
    const uint2 q = *reinterpret_cast<const uint2*>((const bf16_t*)p + i);
    v[0] = __uint_as_float(q.x << 16);
    v[1] = __uint_as_float(q.x & 0xffff0000u);
    v[2] = __uint_as_float(q.y << 16);
    v[3] = __uint_as_float(q.y & 0xffff0000u);
  }
}

// value of lane ^ 1 / lane ^ 2 (DPP quad permutations [1,0,3,2] / [2,3,0,1])
PG_DEV float dpp_xor1(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0xB1, 0xF, 0xF, false));
}
PG_DEV float dpp_xor2(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x4E, 0xF, 0xF, false));
}

// swizzled element offset of (row r, 16-byte chunk c) in a tile of 32-element rows
PG_DEV int sw_off(int r, int c) { return r * 32 + 8 * (c ^ ((r >> 2) & 3)); }

template <int WN, int WM, int TN, int TM, int GATHER, bool RELU>
__global__ __launch_bounds__(256, 2) void k_conv_fwd(CfK k) {
  constexpr int BN = WN * TN * 32, BM = WM * TM * 32;
  constexpr int AP = BM / 64;                  // pixel rows per thread
  constexpr int BP = (BN * 4 + 255) / 256;     // weight chunks per thread
  __shared__ __attribute__((aligned(16))) bf16_t Xs[2][BM * 32];
  __shared__ __attribute__((aligned(16))) bf16_t Ws[2][BN * 32];

  const int bid = remap_tile2(blockIdx.x, k.tiles_m * k.tiles_n);
  const int tmi = bid / k.tiles_n, tni = bid - tmi * k.tiles_n;
  const int m0 = tmi * BM, n0 = tni * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wn = wave / WM, wm = wave % WM;
  const int q = tid & 3;
  const bool quad = k.o.pool;
  const int C = k.C, R = k.R, pad = k.pad;

  int rb[AP], roh[AP], row_[AP];
  bool rv[AP];
#pragma unroll
  for (int p = 0; p < AP; ++p) {
    const int m = m0 + (tid >> 2) + 64 * p;
    rv[p] = m < k.M;
    pix_of(k, rv[p] ? m : 0, quad, rb[p], roh[p], row_[p]);
  }
  // byte offsets of this thread's 16-byte chunks (kOOB: reads zeros)
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(k.x, k.x_bytes);
  const __amdgpu_buffer_rsrc_t wr = make_rsrc(k.w, k.w_bytes);
  uint32_t roff[AP];
  auto set_tap = [&](int tap) {
    const int r = tap / R, s = tap - (tap / R) * R;
#pragma unroll
    for (int p = 0; p < AP; ++p) {
      const int ih = roh[p] + r - pad, iw = row_[p] + s - pad;
      const bool ok = rv[p] && (unsigned)ih < (unsigned)k.H && (unsigned)iw < (unsigned)k.W;
      const int sh = GATHER == G_UP2 ? (ih >> 1) : ih;
      const int sw = GATHER == G_UP2 ? (iw >> 1) : iw;
      roff[p] = ok ? (uint32_t)(((rb[p] * k.Hx + sh) * k.Wx + sw) * C + q * 8) * 2u : kOOB;
    }
  };
  uint32_t woff[BP];
#pragma unroll
  for (int p = 0; p < BP; ++p) {
    const int idx = tid + 256 * p;
    const int n = n0 + (idx >> 2);
    woff[p] = idx < BN * 4 && n < k.Np ? (uint32_t)(n * R * R * C + (idx & 3) * 8) * 2u : kOOB;
  }
  // LDS staging offsets (fixed across steps)
  int xst[AP], wst[BP];
#pragma unroll
  for (int p = 0; p < AP; ++p) xst[p] = sw_off((tid >> 2) + 64 * p, q);
#pragma unroll
  for (int p = 0; p < BP; ++p) {
    const int idx = tid + 256 * p;
    wst[p] = idx < BN * 4 ? sw_off(idx >> 2, idx & 3) : 0;
  }

  uint4 ra[AP], rw[BP];
  int ld_tap = 0, ld_c0 = 0, ld_ks = 0;
  set_tap(0);
  auto load = [&]() {
#pragma unroll
    for (int p = 0; p < AP; ++p) ra[p] = buf_ld16(xr, roff[p] + 2u * ld_c0);
#pragma unroll
    for (int p = 0; p < BP; ++p) rw[p] = buf_ld16(wr, woff[p] + 64u * ld_ks);
    ++ld_ks;
    ld_c0 += 32;
    if (ld_c0 == C) {
      ld_c0 = 0;
      ++ld_tap;
      if (ld_tap < R * R) set_tap(ld_tap);
    }
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int p = 0; p < AP; ++p)
      *reinterpret_cast<uint4*>(&Xs[buf][xst[p]]) = RELU ? relu8_bits(ra[p]) : ra[p];
#pragma unroll
    for (int p = 0; p < BP; ++p)
      if (tid + 256 * p < BN * 4) *reinterpret_cast<uint4*>(&Ws[buf][wst[p]]) = rw[p];
  };

  // operand read offsets: row (tile base + lane%32), chunk 2*kk + lane/32
  const int lr = lane & 31, f = (lr >> 2) & 3, h = lane >> 5;
  const int rd0 = lr * 32 + 8 * ((0 + h) ^ f);
  const int rd1 = lr * 32 + 8 * ((2 + h) ^ f);

  f32x16 acc[TN][TM];
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  load();
  store(0);
  __syncthreads();
  int buf = 0;
  for (int ks = 0; ks < k.ksteps; ++ks) {
    const bool more = ks + 1 < k.ksteps;
    if (more) load();
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const int rd = kk ? rd1 : rd0;
      bf16x8 wv[TN], xv[TM];
#pragma unroll
      for (int i = 0; i < TN; ++i)
        wv[i] = *reinterpret_cast<const bf16x8*>(&Ws[buf][(wn * TN + i) * 32 * 32 + rd]);
#pragma unroll
      for (int j = 0; j < TM; ++j)
        xv[j] = *reinterpret_cast<const bf16x8*>(&Xs[buf][(wm * TM + j) * 32 * 32 + rd]);
#pragma unroll
      for (int i = 0; i < TN; ++i)
#pragma unroll
        for (int j = 0; j < TM; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wv[i], xv[j], acc[i][j], 0, 0, 0);
    }
    if (more) store(buf ^ 1);
    __syncthreads();
    buf ^= 1;
  }

  // ---- epilogue: lane holds channels 8g + 4h + (0..3) of pixel m.
  // Per pixel tile: 32-bit element offsets of the output, mask and residual
  // rows (the host guarantees they fit); per channel group: the bias.
  const ConvOut& o = k.o;
  const float accs = (o.acc_scale ? *o.acc_scale : 1.f) * o.acc_mul;
  int yo[TM], mko[TM], ro[TM];
  bool wr_ok[TM];
#pragma unroll
  for (int j = 0; j < TM; ++j) {
    const int m = m0 + (wm * TM + j) * 32 + lr;
    const bool mv = m < k.M;
    const int mo = quad ? (m >> 2) : m;
    wr_ok[j] = mv && (!quad || (lr & 3) == 0);
    yo[j] = mo * o.yC;
    mko[j] = mo * o.maskC;
    int ridx = mo;
    if (o.res_mode == R_HALF) {
      int bb, oh, ow;
      pix_of(k, mv ? m : 0, false, bb, oh, ow);
      ridx = (bb * (k.H >> 1) + (oh >> 1)) * (k.W >> 1) + (ow >> 1);
    }
    ro[j] = ridx * o.resC;
  }
#pragma unroll
  for (int i = 0; i < TN; ++i) {
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
      const int n = n0 + (wn * TN + i) * 32 + 8 * g4 + 4 * h;
      float bias[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) bias[e] = (o.bias && n + e < o.n_real) ? o.bias[n + e] : 0.f;
      const bool n_ok = n < o.yC;
#pragma unroll
      for (int j = 0; j < TM; ++j) {
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = acc[i][j][4 * g4 + e];
        if (quad) {
          // 2x2 average over the four consecutive rows (lanes) of a window
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float t = v[e] + dpp_xor1(v[e]);
            v[e] = 0.25f * (t + dpp_xor2(t));
          }
        }
        if (!(wr_ok[j] && n_ok)) continue;
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = v[e] * accs + bias[e];
        if (o.mask) {
          float mk[4];
          load4(o.mask, o.mask_f32, mko[j] + n, mk);
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = mk[e] > 0.f ? v[e] : 0.f;
        }
        if (o.res_mode != R_NONE) {
          float rv[4];
          load4(o.res, o.res_f32, ro[j] + n, rv);
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] += o.res_scale * rv[e];
        }
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (n + e >= o.n_real) v[e] = 0.f;
        if (o.y_f32) {
          *reinterpret_cast<float4*>((float*)o.y + (yo[j] + n)) = make_float4(v[0], v[1], v[2], v[3]);
        } else {
          *reinterpret_cast<uint2*>((bf16_t*)o.y + (yo[j] + n)) = make_uint2(f2bf2(v[0], v[1]), f2bf2(v[2], v[3]));
        }
      }
    }
  }
}

template <int WN, int WM, int TN, int TM>
std::string launch_cfg(hipStream_t s, CfK& k, int gather, bool relu) {
  constexpr int BN = WN * TN * 32, BM = WM * TM * 32;
  k.tiles_m = (int)cdiv(k.M, BM);
  k.tiles_n = (int)cdiv(k.Np, BN);
  dim3 grid(k.tiles_m * k.tiles_n), block(256);
#define PG_CF_CASE(G, R_)                                                             \
  if (gather == G && relu == R_) {                                                    \
    hipLaunchKernelGGL((k_conv_fwd<WN, WM, TN, TM, G, R_>), grid, block, 0, s, k);    \
    return "k_conv_fwd<" + std::to_string(BN) + "x" + std::to_string(BM) + "," #G "," #R_ ">"; \
  }
  PG_CF_CASE(G_DIRECT, false)
  PG_CF_CASE(G_DIRECT, true)
  PG_CF_CASE(G_UP2, false)
  PG_CF_CASE(G_UP2, true)
#undef PG_CF_CASE
  throw Error{-2, "conv_fwd: unsupported gather"};
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

}  // namespace

bool conv_fwd_mfma_ok(const ConvIn& in, int H, int W, int R, int Np, const ConvOut& o) {
  if (in.mean || in.gather == G_POOL2 || in.gscale != 1.f) return false;
  const int64_t M = (int64_t)in.B * H * W;
  const int64_t Mo = o.pool ? M / 4 : M;
  const int64_t xs = (int64_t)in.B * in.Hx * in.Wx * in.C;
  const int64_t ws = (int64_t)Np * R * R * in.C;
  const int cmax = std::max({o.yC, o.resC, o.maskC});
  if (M >= (1LL << 31) || xs >= (1LL << 31) || ws >= (1LL << 31) || Mo * cmax >= (1LL << 31)) return false;
  if (2 * xs >= kBufMax || 2 * ws >= kBufMax) return false;
  if (o.yC % 4 || (o.res_mode != R_NONE && o.resC % 4) || (o.mask && o.maskC % 4)) return false;
  if (!aligned16(o.y) || (o.res && !aligned16(o.res)) || (o.mask && !aligned16(o.mask))) return false;
  if (o.pool && o.res_mode == R_HALF) return false;
  if (o.pool && (H % 2 || W % 2)) return false;
  return true;
}

std::string conv_fwd_mfma(hipStream_t s, const ConvIn& in, int H, int W, int R, const void* w, int Np,
                          const ConvOut& out) {
  CfK k;
  k.x = (const bf16_t*)in.x;
  k.w = (const bf16_t*)w;
  k.x_bytes = 2LL * in.B * in.Hx * in.Wx * in.C;
  k.w_bytes = 2LL * Np * R * R * in.C;
  k.Hx = in.Hx;
  k.Wx = in.Wx;
  k.C = in.C;
  k.H = H;
  k.W = W;
  k.R = R;
  k.pad = R / 2;
  k.M = (int)((int64_t)in.B * H * W);
  k.Np = Np;
  k.ksteps = R * R * (in.C / 32);
  k.fdW = make_fastdiv(W);
  k.fdH = make_fastdiv(H);
  k.fdW2 = make_fastdiv(std::max(1, W / 2));
  k.fdH2 = make_fastdiv(std::max(1, H / 2));
  k.o = out;
  if (Np % 128 == 0) return launch_cfg<2, 2, 2, 4>(s, k, in.gather, in.relu);
  if (Np % 96 == 0) return launch_cfg<1, 4, 3, 2>(s, k, in.gather, in.relu);
  if (Np <= 64) return launch_cfg<1, 4, 2, 2>(s, k, in.gather, in.relu);
  return launch_cfg<2, 2, 2, 2>(s, k, in.gather, in.relu);
}

}  // namespace pg
