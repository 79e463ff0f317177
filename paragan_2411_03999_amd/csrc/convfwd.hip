// Implicit-GEMM convolution (forward and data gradient) on gfx950 MFMA for
// the direct, nearest-upsample, stride-2 and sub-pixel gathers with a plain
// or ReLU'd operand.
//
// GEMM: rows = output channels n (the packed weights, K contiguous), columns
// = output pixels m (the im2col of the activation, gathered on the fly), K =
// taps x input channels.  With the weights as the MFMA A operand each lane's
// accumulator holds four consecutive output channels of one pixel.  The
// epilogue (scale, bias, ReLU mask, residual) restages each wave's results
// through LDS so that a lane owns eight consecutive channels of one pixel and
// consecutive lanes walk a pixel's channel run: every store is 16 (bf16) or
// 32 (fp32) contiguous bytes and a wave writes whole cache lines.
//
// K loop: tap-outer, channel-inner; a thread's source offsets are computed
// once per tap and advance by 32 channels per step.  Operand tiles move
// from HBM straight into LDS (buffer loads with an LDS destination: lane l
// of a wave writes 16 bytes at M0 + 16 l, no registers or LDS stores
// involved) through a ring of three stages, so the loads of step k + 2 are
// in flight while step k computes; one barrier per step.  LDS rows are 64
// bytes (32 bf16 of K) with the 16-byte chunks XOR-swizzled by row, which
// keeps the MFMA operand reads free of bank conflicts; the swizzle is
// realised by choosing which source chunk each lane loads.  A ReLU on the
// activation operand is applied to the fragments as they leave LDS.
#include "lds_dma.hpp"
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
  FastDiv fdW, fdH;
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

// conv-grid position (b, oh, ow) of output row m
PG_DEV void pix_of(const CfK& k, int m, int& b, int& oh, int& ow) {
  const int t = (int)fdiv((uint32_t)m, k.fdW);
  ow = m - t * k.W;
  b = (int)fdiv((uint32_t)t, k.fdH);
  oh = t - b * k.H;
}

// eight consecutive values (16-byte aligned bf16 or 32-byte aligned fp32)
PG_DEV void load8(const void* p, bool f32, int i, float* v) {
  if (f32) {
    const float4 a = *reinterpret_cast<const float4*>((const float*)p + i);
    const float4 b = *reinterpret_cast<const float4*>((const float*)p + i + 4);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
  } else {
    const uint4 q = *reinterpret_cast<const uint4*>((const bf16_t*)p + i);
    const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      v[2 * t] = __uint_as_float(w[t] << 16);
      v[2 * t + 1] = __uint_as_float(w[t] & 0xffff0000u);
    }
  }
}

// swizzled element offset of (row r, 16-byte chunk c) in a tile of 32-element rows
PG_DEV int sw_off(int r, int c) { return r * 32 + 8 * (c ^ ((r >> 2) & 3)); }

// One K step of a wave (KS channels): operand fragments of one LDS stage
// through the MFMAs, KS / 16 of them per output tile.
template <int TN, int TM, bool RELU, int KS>
PG_DEV void conv_step(const bf16_t* xs, const bf16_t* ws, int xbase, int wbase, const int (&rdo)[KS / 16],
                      f32x16 (&acc)[TN][TM]) {
#pragma unroll
  for (int kk = 0; kk < KS / 16; ++kk) {
    const int rd = rdo[kk];
    bf16x8 wv[TN], xv[TM];
#pragma unroll
    for (int i = 0; i < TN; ++i) wv[i] = *reinterpret_cast<const bf16x8*>(ws + wbase + i * 32 * KS + rd);
#pragma unroll
    for (int j = 0; j < TM; ++j) {
      if (RELU) {
        const uint4 q = relu8_bits(*reinterpret_cast<const uint4*>(xs + xbase + j * 32 * KS + rd));
        xv[j] = __builtin_bit_cast(bf16x8, q);
      } else {
        xv[j] = *reinterpret_cast<const bf16x8*>(xs + xbase + j * 32 * KS + rd);
      }
    }
#pragma unroll
    for (int i = 0; i < TN; ++i)
#pragma unroll
      for (int j = 0; j < TM; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wv[i], xv[j], acc[i][j], 0, 0, 0);
  }
}

// Epilogue of the conv kernels, 32 pixels of a wave at a time.  The MFMA
// layout (lane l: channels 8 g + 4 (l / 32) + 0..3 of pixel l % 32) goes to
// this wave's fp32 staging rows in LDS; read back, lane l takes chunk c =
// 64 t + l, i.e. the eight channels 8 (c % NQ) .. + 7 of pixel c / NQ.
// Rows are the block's BM = WM TM 32 consecutive output pixels from m0; the
// caller has no LDS reads of its operands left in flight past the first
// barrier here.
template <int WN, int WM, int TN, int TM, int GATHER>
PG_DEV void conv_epilogue(const CfK& k, f32x16 (&acc)[TN][TM], bf16_t* lds, int m0, int n0, int wn, int wm,
                          int wave, int lane, int pa, int pb) {
  constexpr int NW = WN * WM, NT = NW * 64, BN = WN * TN * 32;
  constexpr int SROW = TN * 32 + 4;            // staging floats per pixel row
  const int tid = wave * 64 + lane, lr = lane & 31, h = lane >> 5;
  constexpr int NQ = TN * 4;                   // 8-channel chunks per pixel
  const ConvOut& o = k.o;
  const float accs = (o.acc_scale ? *o.acc_scale : 1.f) * o.acc_mul / (o.acc_div ? *o.acc_div : 1.f);
  float* const stg = reinterpret_cast<float*>(lds) + wave * 32 * SROW;
  // the block's bias, past every wave's staging rows
  float* const bsh = reinterpret_cast<float*>(lds) + NW * 32 * SROW;
  const int nw = n0 + wn * TN * 32;
  const float* const bw = bsh + wn * TN * 32;
  // raw 16-byte words of a mask / residual chunk: bf16 (one word) or fp32 (two)
  auto ld_raw = [](const void* base, bool f32, int i, uint4* w) {
    if (f32) {
      w[0] = *reinterpret_cast<const uint4*>((const float*)base + i);
      w[1] = *reinterpret_cast<const uint4*>((const float*)base + i + 4);
    } else {
      w[0] = *reinterpret_cast<const uint4*>((const bf16_t*)base + i);
    }
  };
  // the mask and residual words of output row m (at output pixel mo), channel n
  auto load_mr = [&](int m, int mo, int n, uint4* mwt, uint4* rwt) {
    if (o.mask) ld_raw(o.mask, o.mask_f32, mo * o.maskC + n, mwt);
    if (o.res_mode != R_NONE) {
      int ridx = mo;
      if (o.res_mode == R_HALF) {
        int bb, oh, ow;
        pix_of(k, m, bb, oh, ow);
        ridx = (bb * (k.H >> 1) + (oh >> 1)) * (k.W >> 1) + (ow >> 1);
      }
      ld_raw(o.res, o.res_f32, ridx * o.resC + n, rwt);
    }
  };
  auto unpack_raw = [](const uint4* w, bool f32, float* v) {
    if (f32) {
      const float4 a = __builtin_bit_cast(float4, w[0]), b = __builtin_bit_cast(float4, w[1]);
      v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
    } else {
      unpack8(w[0], v);
    }
  };
  // up to 12 chunks per pixel (TN <= 3) the mask / residual words of a pass
  // fit in registers beside the accumulators; wider tiles load them in place
  constexpr bool PF = TN <= 3;
#pragma unroll
  for (int j = 0; j < TM; ++j) {
    // this lane's chunks of the pass: output index (-1: none), and the mask
    // and residual words, loaded before the staging barriers so that their
    // latency overlaps the staging
    const int mb = m0 + (wm * TM + j) * 32;
    int yo[NQ / 2];
    uint4 mw[NQ / 2][2], rw[NQ / 2][2];
#pragma unroll
    for (int t = 0; t < NQ / 2; ++t) {
      const int c = 64 * t + lane, p = c / NQ, q = c - p * NQ;
      const int m = mb + p, n = nw + 8 * q;
      yo[t] = -1;
      if (m >= k.M || n >= o.yC) continue;
      int mo = m;
      if (GATHER == G_SUB) {
        // source-grid pixel (b, i, j) -> output pixel (b, 2i + a, 2j + b) of the 2x grid
        int bb, ii, jj;
        pix_of(k, m, bb, ii, jj);
        mo = (bb * 2 * k.H + 2 * ii + pa) * (2 * k.W) + 2 * jj + pb;
      }
      yo[t] = mo * o.yC + n;
      if (PF) load_mr(m, mo, n, mw[t], rw[t]);
    }
    // (first pass: every wave is done with the ring; later: this wave has
    // read back the previous pass)
    __syncthreads();
    if (j == 0)
      for (int t = tid; t < BN; t += NT) bsh[t] = (o.bias && n0 + t < o.n_real) ? o.bias[n0 + t] : 0.f;
#pragma unroll
    for (int i = 0; i < TN; ++i)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4)
        *reinterpret_cast<float4*>(stg + lr * SROW + i * 32 + 8 * g4 + 4 * h) =
            make_float4(acc[i][j][4 * g4], acc[i][j][4 * g4 + 1], acc[i][j][4 * g4 + 2], acc[i][j][4 * g4 + 3]);
    __syncthreads();
#pragma unroll
    for (int t = 0; t < NQ / 2; ++t) {
      if (yo[t] < 0) continue;
      const int c = 64 * t + lane, p = c / NQ, q = c - p * NQ;
      const int n = nw + 8 * q;
      if (!PF) load_mr(mb + p, yo[t] / o.yC, n, mw[t], rw[t]);
      float v[8];
      {
        const float4 a = *reinterpret_cast<const float4*>(stg + p * SROW + 8 * q);
        const float4 b = *reinterpret_cast<const float4*>(stg + p * SROW + 8 * q + 4);
        v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
        v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
      }
      {
        const float4 a = *reinterpret_cast<const float4*>(bw + 8 * q);
        const float4 b = *reinterpret_cast<const float4*>(bw + 8 * q + 4);
        const float bv[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = v[e] * accs + bv[e];
      }
      if (o.mask) {
        float mk[8];
        unpack_raw(mw[t], o.mask_f32, mk);
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = mk[e] > 0.f ? v[e] : 0.f;
      }
      if (o.res_mode != R_NONE) {
        float rv8[8];
        unpack_raw(rw[t], o.res_f32, rv8);
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] += o.res_scale * rv8[e];
      }
      if (n + 8 > o.n_real) {
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (n + e >= o.n_real) v[e] = 0.f;
      }
      if (o.y_f32) {
        float* yp = (float*)o.y + yo[t];
        *reinterpret_cast<float4*>(yp) = make_float4(v[0], v[1], v[2], v[3]);
        *reinterpret_cast<float4*>(yp + 4) = make_float4(v[4], v[5], v[6], v[7]);
      } else {
        *reinterpret_cast<uint4*>((bf16_t*)o.y + yo[t]) =
            make_uint4(f2bf2(v[0], v[1]), f2bf2(v[2], v[3]), f2bf2(v[4], v[5]), f2bf2(v[6], v[7]));
      }
    }
  }
}

template <int WN, int WM, int TN, int TM, int NS, int KS, int GATHER, bool RELU>
__global__ __launch_bounds__(WN * WM * 64, 8 / (WN * WM)) void k_conv_fwd(CfK k) {
  constexpr int NW = WN * WM;                  // waves per block (4 or 8)
  constexpr int NT = NW * 64;
  constexpr int BN = WN * TN * 32, BM = WM * TM * 32;
  static_assert(KS == 32 || KS == 64, "channels per step");
  constexpr int CH = KS / 8;                   // 16-byte chunks per LDS row
  constexpr int RPL = 64 / CH;                 // rows filled by one wave load (1 KB)
  constexpr int RG = RPL * NW;                 // tile rows covered by one load of every wave
  static_assert(BM % RG == 0, "activation rows must be whole block loads");
  constexpr int AP = BM / RG;                  // activation wave loads per wave per step
  constexpr int WR = (BN + RG - 1) / RG * RG;  // weight rows held in LDS (whole block loads)
  constexpr int BP = WR / RG;                  // weight wave loads per wave per step
  constexpr int LPS = AP + BP;                 // loads per wave per step
  static_assert(NS >= 2 && NS <= 6, "ring depth");
  constexpr int RING = NS * (BM + WR) * KS;    // bf16 elements of the operand ring
  constexpr int SROW = TN * 32 + 4;            // epilogue staging: floats per pixel row
  constexpr int STG = NW * 32 * SROW * 2;      // (NW waves x 32 pixels, in bf16 elements)
  constexpr int EPI = STG + 2 * BN;            // staging + the block's bias (fp32)
  __shared__ __attribute__((aligned(16))) bf16_t lds[RING > EPI ? RING : EPI];
  bf16_t(*const Xs)[BM * KS] = reinterpret_cast<bf16_t(*)[BM * KS]>(lds);
  bf16_t(*const Ws)[WR * KS] = reinterpret_cast<bf16_t(*)[WR * KS]>(lds + NS * BM * KS);

  // sub-pixel gather: the parity class (a, b) of this block's output pixels
  // varies fastest, so the four classes of a tile run back to back on one
  // XCD and their interleaved output pixels meet in its L2
  const int lin = remap_tile2(blockIdx.x, k.tiles_m * k.tiles_n * (GATHER == G_SUB ? 4 : 1));
  const int par = GATHER == G_SUB ? (lin & 3) : 0;
  const int bid = GATHER == G_SUB ? (lin >> 2) : lin;
  const int tmi = bid / k.tiles_n, tni = bid - tmi * k.tiles_n;
  const int m0 = tmi * BM, n0 = tni * BN;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wn = wave / WM, wm = wave % WM;
  const int pa = par >> 1, pb = par & 1;
  const int C = k.C, R = k.R, pad = k.pad;

  // Load j of this wave covers tile rows RPL (NW j + wave) .. + RPL - 1;
  // lane l fills row + l / CH, LDS chunk l % CH, which in the swizzled
  // layout holds source chunk (l % CH) ^ swz(row): rows of 64 bytes swizzle
  // by (row / 4) % 4, rows of 128 bytes by (row / 2) % 8 (bits of the row
  // that a load's base, a multiple of RPL, leaves alone apart from bit 3,
  // whose value -- the parity of NW j + wave -- is that of wave).
  const int lrow = lane / CH;
  const int lrow_all = RPL * wave + lrow;      // row of load 0 (same swizzle for every load)
  const uint32_t lchunk =
      (uint32_t)((lane % CH) ^ (KS == 32 ? ((lrow_all >> 2) & 3) : ((lrow_all >> 1) & 7)));
  int rb[AP], roh[AP], row_[AP];
  bool rv[AP];
#pragma unroll
  for (int j = 0; j < AP; ++j) {
    const int m = m0 + RPL * (NW * j + wave) + lrow;
    rv[j] = m < k.M;
    pix_of(k, rv[j] ? m : 0, rb[j], roh[j], row_[j]);
  }
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(k.x, k.x_bytes);
  const __amdgpu_buffer_rsrc_t wr = make_rsrc(k.w, k.w_bytes);
  uint32_t roff[AP];
  auto set_tap = [&](int tap) {
    const int r = tap / R, s = tap - (tap / R) * R;
#pragma unroll
    for (int j = 0; j < AP; ++j) {
      // source row / column: the conv-grid position plus the tap (twice the
      // position for the stride-2 gather, whose source is twice the grid)
      const int ih = GATHER == G_S2 ? 2 * roh[j] + r - pad : (GATHER == G_SUB ? roh[j] + r - 1 + pa : roh[j] + r - pad);
      const int iw = GATHER == G_S2 ? 2 * row_[j] + s - pad : (GATHER == G_SUB ? row_[j] + s - 1 + pb : row_[j] + s - pad);
      const int hb = GATHER == G_S2 ? k.Hx : k.H, wb = GATHER == G_S2 ? k.Wx : k.W;
      const bool ok = rv[j] && (unsigned)ih < (unsigned)hb && (unsigned)iw < (unsigned)wb;
      const int sh = GATHER == G_UP2 ? (ih >> 1) : ih;
      const int sw = GATHER == G_UP2 ? (iw >> 1) : iw;
      roff[j] = ok ? (uint32_t)(((rb[j] * k.Hx + sh) * k.Wx + sw) * C) * 2u + 16u * lchunk : kOOB;
    }
  };
  uint32_t woff[BP];
#pragma unroll
  for (int j = 0; j < BP; ++j) {
    const int row = RPL * (NW * j + wave) + lrow;
    const int n = n0 + row;
    // (the sub-pixel gather keeps one filter per parity, [4][Np][2][2][C])
    woff[j] = row < BN && n < k.Np ? (uint32_t)((par * k.Np + n) * R * R * C) * 2u + 16u * lchunk : kOOB;
  }

  // producer position (tap, channel offset, step)
  int ld_tap = 0, ld_c0 = 0, ld_ks = 0;
  set_tap(0);
  auto advance = [&]() {
    ++ld_ks;
    ld_c0 += KS;
    if (ld_c0 == C) {
      ld_c0 = 0;
      ++ld_tap;
      if (ld_tap < R * R) set_tap(ld_tap);
    }
  };
  // LDS bases of this wave's loads in stage 0 (stage s adds s * stage size)
  const uint32_t xl0 = lds_addr(&Xs[0][RPL * wave * KS]), wl0 = lds_addr(&Ws[0][RPL * wave * KS]);
  auto issue = [&](int stage) {
    const uint32_t coff = __builtin_amdgcn_readfirstlane(2u * (uint32_t)ld_c0);
    const uint32_t wk = __builtin_amdgcn_readfirstlane(2u * KS * (uint32_t)ld_ks);
    const uint32_t xl = xl0 + (uint32_t)stage * (BM * KS * 2), wl = wl0 + (uint32_t)stage * (WR * KS * 2);
#pragma unroll
    for (int j = 0; j < AP; ++j) lds_load16(xl + j * (NW * 1024u), roff[j], coff, xr);
#pragma unroll
    for (int j = 0; j < BP; ++j) lds_load16(wl + j * (NW * 1024u), woff[j], wk, wr);
    advance();
  };

  // operand read offsets: row (tile base + lane%32), chunk 2*kk + lane/32
  const int lr = lane & 31, h = lane >> 5;
  const int f = KS == 32 ? ((lr >> 2) & 3) : ((lr >> 1) & 7);
  int rdo[KS / 16];
#pragma unroll
  for (int kk = 0; kk < KS / 16; ++kk) rdo[kk] = lr * KS + 8 * ((2 * kk + h) ^ f);
  const int xbase = wm * TM * 32 * KS, wbase = wn * TN * 32 * KS;

  f32x16 acc[TN][TM];
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int ksteps = k.ksteps;
  // Ring of NS stages: the loads of step s go to stage s % NS and are issued
  // NS - 1 steps ahead.  Step ks first waits until its own loads have landed
  // (those of the up to NS - 2 later steps may still fly) and this wave's
  // reads of step ks - 1 are done, then barriers: past it every wave's loads
  // of step ks are visible and no wave still reads stage (ks - 1) % NS, which
  // it refills with step ks + NS - 1.
#pragma unroll
  for (int s = 0; s < NS - 1; ++s)
    if (s < ksteps) issue(s);
  int ks = 0;
  // steady state, NS steps per trip with compile-time stages (constant LDS
  // addresses), every step refilling a stage
  for (; ks + 2 * NS - 2 < ksteps; ks += NS) {
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      wait_barrier<vm_cap((NS - 2) * LPS)>();
      issue((s + NS - 1) % NS);
      conv_step<TN, TM, RELU, KS>(Xs[s], Ws[s], xbase, wbase, rdo, acc);
    }
  }
  // drain: at most 2 NS - 2 steps, the last NS - 1 of them issuing nothing
  for (; ks < ksteps; ++ks) {
    const int st = ks % NS;
    wait_barrier_steps<LPS>(min(NS - 2, ksteps - 1 - ks));
    if (ks + NS - 1 < ksteps) issue((st + NS - 1) % NS);
    conv_step<TN, TM, RELU, KS>(Xs[st], Ws[st], xbase, wbase, rdo, acc);
  }

  conv_epilogue<WN, WM, TN, TM, GATHER>(k, acc, lds, m0, n0, wn, wm, wave, lane, pa, pb);
}

// Halo variant for the 3x3, pad-1 convolution over the direct gather
// (GK = G_DIRECT, nine taps) and for the sub-pixel gather (GK = G_SUB, the
// four 2x2 taps of one parity class over the source grid), used when a
// block tile is TR = BM / W whole image rows of one image.  The loop runs
// over 32-channel chunks outside and the T taps inside: per chunk, the
// tile's rows plus a one-pixel border -- a (TR + 2) x (W + 2) patch -- move
// into LDS once (double-buffered, the next chunk's patch issued at the
// chunk's first tap), and every tap reads its operand rows out of the patch
// at its offset, so the activation crosses the load path once per chunk
// instead of once per tap.  The weights of each tap step come through a
// ring of NSW stages as in k_conv_fwd; T is a multiple of NSW, so the stage
// of tap t is t % NSW.  Patch rows keep the 64-byte row layout and swizzle
// of k_conv_fwd, indexed by patch pixel.
// compile-time loop: f(std::integral_constant<int, I>) for I = B .. E - 1
template <int B, int E, typename F>
PG_DEV void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

template <int WN, int WM, int TN, int TM, int PPX, int GK, bool RELU>
__global__ __launch_bounds__(WN * WM * 64, 8 / (WN * WM)) void k_conv_halo(CfK k) {
  static_assert(GK == G_DIRECT || GK == G_SUB || GK == G_S2, "halo gathers");
  // Chunks: 32 channels of the source (direct, sub-pixel), or for the
  // stride-2 4x4 filter 32 channels of one parity class (a, b) of the
  // source pixels (2i + a, 2j + b) -- chunk c: slice c / 4, class c % 4 --
  // a 2x2 conv over that class with the taps (2 dr + 1 - a, 2 ds + 1 - b).
  constexpr int T = GK == G_DIRECT ? 9 : 4;    // taps per chunk
  // weight ring stages of one tap each: each tap's weights are issued two
  // steps ahead (measured: for the four-tap sub-pixel chunks, two stages
  // leave the waits exposed; deeper rings gain nothing on the nine-tap ones)
  constexpr int NSW = 3;
  constexpr int NW = WN * WM;
  constexpr int BN = WN * TN * 32, BM = WM * TM * 32;
  constexpr int RG = 16 * NW;                  // rows covered by one load of every wave
  constexpr int WR = (BN + RG - 1) / RG * RG, BP = WR / RG;
  static_assert(PPX % RG == 0, "patch rows are whole block loads");
  constexpr int PLW = PPX / RG;                // patch loads per wave per chunk
  constexpr int PATCH = PPX * 32, WST = WR * 32;   // bf16 elements
  constexpr int RING = 2 * PATCH + NSW * WST;
  constexpr int SROW = TN * 32 + 4;
  constexpr int EPI = NW * 32 * SROW * 2 + 2 * BN;
  __shared__ __attribute__((aligned(16))) bf16_t lds[RING > EPI ? RING : EPI];

  // sub-pixel gather: parity class fastest (as in k_conv_fwd)
  const int lin = remap_tile2(blockIdx.x, k.tiles_m * k.tiles_n * (GK == G_SUB ? 4 : 1));
  const int par = GK == G_SUB ? (lin & 3) : 0;
  const int bid = GK == G_SUB ? (lin >> 2) : lin;
  const int tmi = bid / k.tiles_n, tni = bid - tmi * k.tiles_n;
  const int m0 = tmi * BM, n0 = tni * BN;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wn = wave / WM, wm = wave % WM;
  const int pa = par >> 1, pb = par & 1;
  const int C = k.C, H = k.H, W = k.W, PC = W + 2;
  // the tile: rows tr0 .. tr0 + TR - 1 of image b (the host checks that W
  // divides BM and BM / W divides H)
  const int TR = BM / W;
  const int t0 = (int)fdiv((uint32_t)m0, k.fdW);
  const int b = (int)fdiv((uint32_t)t0, k.fdH), tr0 = t0 - b * H;
  const int npx = (TR + 2) * PC;

  // loads: load j of this wave covers rows 16 (NW j + wave) .. + 15 of the
  // patch (pixels) or of the weight tile; lane l fills row + l / 4, LDS
  // chunk l % 4 = source chunk (l % 4) ^ ((l / 16) % 4)
  const int lrow = lane >> 2;
  const uint32_t lchunk = (uint32_t)((lane & 3) ^ ((lane >> 4) & 3));
  uint32_t poff[PLW];
#pragma unroll
  for (int j = 0; j < PLW; ++j) {
    const int q = 16 * (NW * j + wave) + lrow;
    const int pr = q / PC, pc = q - pr * PC;
    const int ih = tr0 - 1 + pr, iw = pc - 1;
    const bool ok = q < npx && (unsigned)ih < (unsigned)H && (unsigned)iw < (unsigned)W;
    // (stride 2: the class (0, 0) pixel of the source's 2x2 window; the
    // chunk's class adds its offset)
    const int pix = GK == G_S2 ? (b * k.Hx + 2 * ih) * k.Wx + 2 * iw : (b * H + ih) * W + iw;
    poff[j] = ok ? (uint32_t)(pix * C) * 2u + 16u * lchunk : kOOB;
  }
  uint32_t woff[BP];
#pragma unroll
  for (int j = 0; j < BP; ++j) {
    const int row = 16 * (NW * j + wave) + lrow;
    const int n = n0 + row;
    // (the sub-pixel filters are [4][Np][2][2][C], one per parity; the
    // stride-2 ones [Np][4][4][C])
    const int wrow = GK == G_S2 ? n * 16 : (par * k.Np + n) * T;
    woff[j] = row < BN && n < k.Np ? (uint32_t)(wrow * C) * 2u + 16u * lchunk : kOOB;
  }
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(k.x, k.x_bytes);
  const __amdgpu_buffer_rsrc_t wr = make_rsrc(k.w, k.w_bytes);
  const uint32_t pl0 = lds_addr(lds + 16 * wave * 32), wl0 = lds_addr(lds + 2 * PATCH + 16 * wave * 32);
  // chunk c's patch into buffer buf
  auto issue_patch = [&](int buf, int c) {
    const uint32_t coff = __builtin_amdgcn_readfirstlane(
        GK == G_S2 ? 64u * (uint32_t)(c >> 2) + (uint32_t)((((c >> 1) & 1) * k.Wx + (c & 1)) * C) * 2u
                   : 64u * (uint32_t)c);
    const uint32_t pl = pl0 + (uint32_t)buf * (PATCH * 2);
#pragma unroll
    for (int j = 0; j < PLW; ++j) lds_load16(pl + j * (NW * 1024u), poff[j], coff, xr);
  };
  // weights of step s (chunk s / T, tap s % T) into stage st
  auto issue_w = [&](int st, int step) {
    const int c = step / T, t = step - T * c;
    // stride 2: tap (r, s) = (2 dr + 1 - a, 2 ds + 1 - b) of the 4x4 filter
    const int wtap = GK == G_S2 ? (2 * (t >> 1) + 1 - ((c >> 1) & 1)) * 4 + 2 * (t & 1) + 1 - (c & 1) : t;
    const int wch = GK == G_S2 ? 32 * (c >> 2) : 32 * c;
    const uint32_t wk = __builtin_amdgcn_readfirstlane(2u * (uint32_t)(wtap * C + wch));
    const uint32_t wl = wl0 + (uint32_t)st * (WST * 2);
#pragma unroll
    for (int j = 0; j < BP; ++j) lds_load16(wl + j * (NW * 1024u), woff[j], wk, wr);
  };

  // operand reads: weight rows as in k_conv_fwd; activation fragment j of
  // this wave holds tile pixels p = (wm TM + j) 32 + lane % 32, read at
  // patch pixel q0 + r PC + s for tap offset (r, s), q0 = (p / W) PC + p % W
  // (direct: tap t at (t / 3, t % 3); sub-pixel: (t / 2 + a, t % 2 + b))
  const int lr = lane & 31, h = lane >> 5;
  const int f = (lr >> 2) & 3;
  const int rdw[2] = {lr * 32 + 8 * ((0 + h) ^ f), lr * 32 + 8 * ((2 + h) ^ f)};
  const int wbase = wn * TN * 32 * 32;
  int q0[TM];
#pragma unroll
  for (int j = 0; j < TM; ++j) {
    const int p = (wm * TM + j) * 32 + lr;
    const int ty = (int)fdiv((uint32_t)p, k.fdW);
    q0[j] = ty * PC + (p - ty * W);
  }

  f32x16 acc[TN][TM];
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // Issue order: P(0) W(0) .. W(NSW - 2), then at step s W(s + NSW - 1)
  // and, at a chunk's first tap, P(c + 1).  Step s waits until W(s) -- and
  // with it every earlier load, P(c) among them -- has landed; still in
  // flight may be W(s + 1) .. W(s + NSW - 2) (those that exist) and, at taps
  // 1 .. NSW - 1, P(c + 1).  The barrier then also guarantees that no wave
  // reads weight stage (s - 1) % NSW or patch buffer (c + 1) % 2 (last read
  // in chunk c - 1) any more before they refill.
  static_assert(NSW >= 2 && NSW <= T, "the next patch is issued within a chunk");
  const int nch = (GK == G_S2 ? 4 : 1) * (C / 32), S = T * nch;
  issue_patch(0, 0);
#pragma unroll
  for (int st = 0; st < NSW - 1; ++st)
    if (st < S) issue_w(st, st);
  int sb = 0;   // ring stage of the chunk's first tap, (T c) % NSW
  for (int c = 0; c < nch; ++c) {
    const bf16_t* Pc = lds + (c & 1) * PATCH;
    const bool more = c + 1 < nch;
    // the patch offset of tap (dr, ds) is (dr + ca) PC + ds + cb
    const int ca = GK == G_S2 ? 1 - ((c >> 1) & 1) : pa, cb = GK == G_S2 ? 1 - (c & 1) : pb;
    // activation fragments (both 16-channel halves) of tap t at patch offset qo
    auto read_x = [&](int qo, uint4 (&xr)[2][TM]) {
#pragma unroll
      for (int kk = 0; kk < 2; ++kk)
#pragma unroll
        for (int j = 0; j < TM; ++j) {
          const int q = q0[j] + qo;
          xr[kk][j] = *reinterpret_cast<const uint4*>(Pc + q * 32 + 8 * ((2 * kk + h) ^ ((q >> 2) & 3)));
        }
    };
    auto tap_off = [&](int t) {
      return GK != G_DIRECT ? ((t >> 1) + ca) * PC + (t & 1) + cb : (t / 3) * PC + (t % 3);
    };
    // Per tap: all operand reads first, then the MFMAs (the compiler would
    // otherwise interleave them two by two, waiting on each read).  The
    // activation fragments of the next tap of the chunk come from the same
    // patch buffer, which no load touches during the chunk, so they are read
    // as soon as this tap's MFMAs are issued, ahead of the next barrier;
    // after it only the weight reads are left.
    uint4 xnext[2][TM];
    static_for<0, T>([&](auto tc) {
      constexpr int t = decltype(tc)::value;
      constexpr int wfly = (NSW - 2) * BP + (t >= 1 && t <= NSW - 1 ? PLW : 0);
      constexpr int wlast = (NSW - 2 < T - 1 - t ? NSW - 2 : T - 1 - t) * BP;
      const int s = T * c + t;
      if (more) wait_barrier<vm_cap(wfly)>();
      else wait_barrier<vm_cap(wlast)>();
      if (s + NSW - 1 < S) issue_w((sb + t + NSW - 1) % NSW, s + NSW - 1);
      if (t == 0 && more) issue_patch((c + 1) & 1, c + 1);
      const bf16_t* Wt = lds + 2 * PATCH + ((sb + t) % NSW) * WST;
      bf16x8 wv[2][TN];
      uint4 xr[2][TM];
#pragma unroll
      for (int kk = 0; kk < 2; ++kk)
#pragma unroll
        for (int i = 0; i < TN; ++i) wv[kk][i] = *reinterpret_cast<const bf16x8*>(Wt + wbase + i * 32 * 32 + rdw[kk]);
      if (t == 0) read_x(tap_off(0), xr);
      else {
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
          for (int j = 0; j < TM; ++j) xr[kk][j] = xnext[kk][j];
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        bf16x8 xv[TM];
#pragma unroll
        for (int j = 0; j < TM; ++j) xv[j] = __builtin_bit_cast(bf16x8, RELU ? relu8_bits(xr[kk][j]) : xr[kk][j]);
#pragma unroll
        for (int i = 0; i < TN; ++i)
#pragma unroll
          for (int j = 0; j < TM; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wv[kk][i], xv[j], acc[i][j], 0, 0, 0);
      }
      if (t + 1 < T) read_x(tap_off(t + 1), xnext);
    });
    sb = (sb + T) % NSW;
  }
  conv_epilogue<WN, WM, TN, TM, GK == G_SUB ? G_SUB : G_DIRECT>(k, acc, lds, m0, n0, wn, wm, wave, lane, pa, pb);
}

template <int WN, int WM, int TN, int TM, int PPX, int GK>
std::string launch_halo(hipStream_t s, CfK& k, bool relu) {
  constexpr int BN = WN * TN * 32, BM = WM * TM * 32;
  k.tiles_m = (int)cdiv(k.M, BM);
  k.tiles_n = (int)cdiv(k.Np, BN);
  k.ksteps = (GK == G_DIRECT ? 9 : GK == G_S2 ? 16 : 4) * (k.C / 32);
  dim3 grid(k.tiles_m * k.tiles_n * (GK == G_SUB ? 4 : 1)), block(64 * WN * WM);
  const std::string name = "k_conv_halo<" + std::to_string(BN) + "x" + std::to_string(BM) +
                           (GK == G_SUB ? ",G_SUB" : GK == G_S2 ? ",G_S2" : "") + (relu ? ",true>" : ",false>");
  if constexpr (GK != G_SUB) {
    if (relu)
      hipLaunchKernelGGL((k_conv_halo<WN, WM, TN, TM, PPX, GK, true>), grid, block, 0, s, k);
    else
      hipLaunchKernelGGL((k_conv_halo<WN, WM, TN, TM, PPX, GK, false>), grid, block, 0, s, k);
  } else {
    if (relu) throw Error{-2, "conv_fwd: no ReLU'd operand for the sub-pixel gather"};
    hipLaunchKernelGGL((k_conv_halo<WN, WM, TN, TM, PPX, GK, false>), grid, block, 0, s, k);
  }
  return name;
}
// patch pixels of a BM-pixel tile of whole rows of a W-wide image (0: not eligible)
inline int halo_patch(int BM, int H, int W) {
  if (W < 16 || BM % W || H % (BM / W)) return 0;
  return (BM / W + 2) * (W + 2);
}

template <int WN, int WM, int TN, int TM, int NS = 3, int KS = 32>
std::string launch_cfg(hipStream_t s, CfK& k, int gather, bool relu) {
  constexpr int BN = WN * TN * 32, BM = WM * TM * 32;
  if (k.C % KS) throw Error{-2, "conv_fwd: channels per step"};
  k.ksteps = k.R * k.R * (k.C / KS);
  k.tiles_m = (int)cdiv(k.M, BM);
  k.tiles_n = (int)cdiv(k.Np, BN);
  dim3 grid(k.tiles_m * k.tiles_n * (gather == G_SUB ? 4 : 1)), block(64 * WN * WM);
#define PG_CF_CASE(G, R_)                                                             \
  if (gather == G && relu == R_) {                                                    \
    hipLaunchKernelGGL((k_conv_fwd<WN, WM, TN, TM, NS, KS, G, R_>), grid, block, 0, s, k); \
    return "k_conv_fwd<" + std::to_string(BN) + "x" + std::to_string(BM) + (KS == 32 ? "" : "k" + std::to_string(KS)) + \
           (NS == 3 ? "" : "/" + std::to_string(NS)) + "," #G "," #R_ ">"; \
  }
  PG_CF_CASE(G_DIRECT, false)
  PG_CF_CASE(G_DIRECT, true)
  PG_CF_CASE(G_UP2, false)
  PG_CF_CASE(G_UP2, true)
  PG_CF_CASE(G_S2, false)
  PG_CF_CASE(G_S2, true)
  PG_CF_CASE(G_SUB, false)
#undef PG_CF_CASE
  throw Error{-2, "conv_fwd: unsupported gather"};
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

}  // namespace

bool conv_fwd_mfma_ok(const ConvIn& in, int H, int W, int R, int Np, const ConvOut& o) {
  if (in.mean || in.gather == G_POOL2 || in.gscale != 1.f) return false;
  const int64_t M = (int64_t)in.B * H * W;
  const int64_t Mo = M;
  const int64_t xs = (int64_t)in.B * in.Hx * in.Wx * in.C;
  const int64_t ws = (int64_t)Np * R * R * in.C;
  const int cmax = std::max({o.yC, o.resC, o.maskC});
  if (M >= (1LL << 31) || xs >= (1LL << 31) || ws >= (1LL << 31) || Mo * cmax >= (1LL << 31)) return false;
  if (2 * xs >= kBufMax || 2 * ws >= kBufMax) return false;
  // (the epilogue moves 8-channel runs; 2x2 pooling is left to the general kernel)
  if (o.pool || o.yC % 8 || (o.res_mode != R_NONE && o.resC % 8) || (o.mask && o.maskC % 8)) return false;
  if (!aligned16(o.y) || (o.res && !aligned16(o.res)) || (o.mask && !aligned16(o.mask))) return false;
  if (in.gather == G_S2 && ((R != 4 && R != 2) || in.Hx != 2 * H || in.Wx != 2 * W)) return false;
  if (in.gather == G_SUB &&
      (R != 2 || in.relu || in.Hx != H || in.Wx != W || o.res_mode != R_NONE || 4 * Mo * cmax >= (1LL << 31)))
    return false;
  return true;
}

std::string conv_fwd_mfma(hipStream_t s, const ConvIn& in, int H, int W, int R, const void* w, int Np,
                          const ConvOut& out) {
  CfK k;
  k.x = (const bf16_t*)in.x;
  k.w = (const bf16_t*)w;
  k.x_bytes = 2LL * in.B * in.Hx * in.Wx * in.C;
  k.w_bytes = 2LL * Np * R * R * in.C * (in.gather == G_SUB ? 4 : 1);
  k.Hx = in.Hx;
  k.Wx = in.Wx;
  k.C = in.C;
  k.H = H;
  k.W = W;
  k.R = R;
  k.pad = in.gather == G_S2 ? (R - 2) / 2 : R / 2;
  k.M = (int)((int64_t)in.B * H * W);
  k.Np = Np;
  k.ksteps = R * R * (in.C / 32);
  k.fdW = make_fastdiv(W);
  k.fdH = make_fastdiv(H);
  k.o = out;
  // Tile choice (measured on the BigGAN shapes in the train step).  For
  // multiples of 256 channels an eight-wave block (one per CU) on a 256 x
  // 256 tile halves the operand bytes per MFMA of the four-wave 128 x 256
  // tile, and wins whenever its blocks come in whole rounds over the CUs
  // (the last round at least three quarters full); with a ragged last round
  // the four-wave tiles, two per CU, spread better.  Otherwise: 128 x 256
  // for multiples of 128 (128 x 128 for exactly 128, the 1x1 attention
  // projections with K <= 192), 192 x 128 for multiples of 192, 96 x 256
  // for the other multiples of 96, and 32 / 64 x 256 for narrow outputs.
  // Direct 3x3 convs whose tiles are whole image rows take the halo kernel
  // (each activation chunk loaded once for all nine taps) on the 256 x 256
  // and 192 x 128 tiles, and for 96 channels on an eight-wave 96 x 512 tile,
  // whose weight loads the wider tile amortises (measured: on the four-wave
  // 128 x 256 tile the patch addressing of its four pixel fragments costs
  // more than the loads it saves).
  const bool halo = in.gather == G_DIRECT && R == 3;
  auto fits = [&](int bm, int ppx) {
    const int np = halo_patch(bm, H, W);
    return halo && np > 0 && np <= ppx;
  };
  const int64_t tiles8 = cdiv(k.M, 256) * (Np / 256) * (in.gather == G_SUB ? 4 : 1);
  const int64_t last8 = tiles8 % 256;
  if (Np % 256 == 0 && tiles8 >= 192 && (last8 == 0 || last8 >= 192))
    return fits(256, 384) ? launch_halo<2, 4, 4, 2, 384, G_DIRECT>(s, k, in.relu)
                          : launch_cfg<2, 4, 4, 2>(s, k, in.gather, in.relu);
  if (Np % 192 == 0 && fits(128, 320)) return launch_halo<2, 2, 3, 2, 320, G_DIRECT>(s, k, in.relu);
  if (Np == 96 && fits(512, 896)) return launch_halo<1, 8, 3, 2, 896, G_DIRECT>(s, k, in.relu);
  // sub-pixel convs (a 2x2 filter per parity over the source grid) share the
  // patch logic, over a 96 x 256 tile and, for multiples of 192 with K = 4 C
  // of at least 768, a 192 x 128 one (measured: 3-7% faster than the ring
  // kernel's tiles on the BigGAN shapes down to that K)
  const bool hsub = in.gather == G_SUB && R == 2;
  auto fits_sub = [&](int bm, int ppx) {
    const int np = halo_patch(bm, H, W);
    return hsub && np > 0 && np <= ppx;
  };
  if (Np % 192 == 0 && in.C >= 192 && fits_sub(128, 320))
    return launch_halo<2, 2, 3, 2, 320, G_SUB>(s, k, false);
  if (Np == 96 && fits_sub(256, 448)) return launch_halo<1, 4, 3, 2, 448, G_SUB>(s, k, false);
  // the stride-2 4x4 filter (pooled D conv2): a patch per parity class of the source
  const bool hs2 = in.gather == G_S2 && R == 4;
  auto fits_s2 = [&](int bm, int ppx) {
    const int np = halo_patch(bm, H, W);
    return hs2 && np > 0 && np <= ppx;
  };
  if (Np % 192 == 0 && fits_s2(128, 320)) return launch_halo<2, 2, 3, 2, 320, G_S2>(s, k, in.relu);
  if (Np == 96 && fits_s2(256, 448)) return launch_halo<1, 4, 3, 2, 448, G_S2>(s, k, in.relu);
  // eight waves on 192 x 256 where those tiles come in whole rounds over
  // the CUs and the four-wave tiles would not
  if (Np % 192 == 0) {
    const int64_t t6 = cdiv(k.M, 256) * (Np / 192) * (in.gather == G_SUB ? 4 : 1), l6 = t6 % 256;
    const int64_t t4 = cdiv(k.M, Np % 128 == 0 ? 256 : 128) * (Np % 128 == 0 ? Np / 128 : Np / 192) *
                       (in.gather == G_SUB ? 4 : 1), l4 = t4 % 512;
    if (t6 >= 192 && (l6 == 0 || l6 >= 192) && l4 != 0 && l4 < 384) return launch_cfg<2, 4, 3, 2>(s, k, in.gather, in.relu);
  }
  if (Np == 128) return launch_cfg<2, 2, 2, 2>(s, k, in.gather, in.relu);
  if (Np % 128 == 0) return launch_cfg<2, 2, 2, 4>(s, k, in.gather, in.relu);
  if (Np % 192 == 0) return launch_cfg<2, 2, 3, 2>(s, k, in.gather, in.relu);
  if (Np % 96 == 0) return launch_cfg<1, 4, 3, 2>(s, k, in.gather, in.relu);
  if (Np <= 32) return launch_cfg<1, 4, 1, 2>(s, k, in.gather, in.relu);
  if (Np <= 64) return launch_cfg<1, 4, 2, 2>(s, k, in.gather, in.relu);
  return launch_cfg<2, 2, 2, 2>(s, k, in.gather, in.relu);
}

}  // namespace pg
