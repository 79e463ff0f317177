// bf16 convolution weight gradients on gfx950 MFMA through LDS transpose reads.
//
//   dW[n][(r, s, c)] = sum over conv-grid pixels m of dY[m][n] * X~[m][(r, s, c)]
//
// where X~ is the im2col view of the activation (direct, a nearest 2x
// upsample of a half-resolution tensor, or read at stride 2 for a 4x4 filter
// over a tensor of twice the grid's size; optionally ReLU'd) and dY the
// output gradient (direct, a nearest 2x upsample of a half-resolution
// gradient, or one parity class (2i + a, 2j + b) of a double-resolution
// gradient: the sub-pixel form of a 3x3 conv over a 2x upsample, see
// wgrad_sub).
// The reduction runs over pixels, which are the rows of both operands in
// memory, so each MFMA operand is a transposed tile.  Here both tiles are
// copied row-major into LDS unchanged (16-byte loads and stores) and the
// transposition happens in the LDS read: ds_read_b64_tr_b16 hands each lane
// four values of one column from four consecutive rows, and two such reads
// form the eight-deep K slice of a v_mfma_f32_32x32x16_bf16 operand.
//
// LDS rows are swizzled in 64-byte blocks so that the 32 lanes of one
// transpose read (four rows x 64 bytes) hit distinct banks of the 64-bank
// LDS.  The pixel range is split over blocks; each split writes its own
// partial sum and the splits are added in a fixed order (bitwise
// reproducible, no float atomics).
#include "ops.hpp"

namespace pg {

namespace {

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

constexpr int kMS = 32;   // pixels per pipeline stage (two MFMA K steps)

// block swizzle of LDS row r for a row of NB 64-byte blocks: for four
// consecutive rows the XOR puts their 64-byte spans on distinct banks
template <int NB>
PG_DEV int swz(int r) {
  return NB % 4 == 0 ? (r & 3) : (NB % 4 == 2 ? ((r >> 1) & 1) : 0);
}
// element offset of (row r, element e) in a swizzled tile of P-element rows
template <int P>
PG_DEV int lds_off(int r, int e) {
  constexpr int NB = P / 32;
  return r * P + ((((e >> 5) ^ swz<NB>(r)) << 5) | (e & 31));
}

// Two transpose reads: 8 consecutive rows (the K slice) of one column.
PG_DEV bf16x8 tr_pair(const bf16_t* base, int off_lo, int off_hi) {
  const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(base + off_lo));
  const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(base + off_hi));
  const auto v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_bit_cast(bf16x8, v);
}

// One 32-deep K step of a wave's TM x TN accumulator tiles: A rows from the
// gradient tile gb (row stride sa), B rows from the activation tile xb (row
// stride sb), both read transposed.  With at most eight tiles every operand
// of the step is read before the first MFMA (left to itself the compiler
// interleaves reads and MFMAs two by two, waiting on each read); wider
// tiles have no registers for that and take each 16-deep half in turn.
template <int TM, int TN>
PG_DEV void wg_step(const bf16_t* gb, const bf16_t* xb, const int (&a_off)[TM], const int (&b_off)[TN], int sa,
                    int sb, f32x16 (&acc)[TM][TN]) {
  if constexpr (TM * TN <= 8) {
    bf16x8 av[2][TM], bv[2][TN];
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
#pragma unroll
      for (int i = 0; i < TM; ++i) av[kk][i] = tr_pair(gb, a_off[i] + kk * 16 * sa, a_off[i] + (kk * 16 + 4) * sa);
#pragma unroll
      for (int j = 0; j < TN; ++j) bv[kk][j] = tr_pair(xb, b_off[j] + kk * 16 * sb, b_off[j] + (kk * 16 + 4) * sb);
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[kk][i], bv[kk][j], acc[i][j], 0, 0, 0);
  } else {
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      bf16x8 av[TM], bv[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) av[i] = tr_pair(gb, a_off[i] + kk * 16 * sa, a_off[i] + (kk * 16 + 4) * sa);
#pragma unroll
      for (int j = 0; j < TN; ++j) bv[j] = tr_pair(xb, b_off[j] + kk * 16 * sb, b_off[j] + (kk * 16 + 4) * sb);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[i], bv[j], acc[i][j], 0, 0, 0);
    }
  }
}

struct WgTrK {
  const bf16_t* g;   // gradient source, channel stride gC
  const bf16_t* x;   // activation source [B][Hx][Wx][C]
  int64_t g_bytes, x_bytes;
  int gC, Np, Kdim, C, R, pad;
  int H, W;          // conv grid
  int Hx, Wx;        // activation source dims
  int Hs, Ws;        // gradient source dims (upsampled gradient)
  int M;             // conv-grid pixels
  FastDiv fdW, fdH, fdC, fdR;
  int m_per_split, tiles_n, tiles_k, splits;
  float scale;       // applied to the sums written (1 when splits are reduced later)
  float* part;       // [splits][Np][Kdim]; parity mode: [4][splits][Np][Kdim]
};

// gradient operand modes
constexpr int kGDirect = 0, kGUp2 = 1, kGParity = 2;

PG_DEV int remap_block(int bid, int total) {
  // Blocks go round-robin to the 8 XCDs; give each XCD a contiguous run of
  // the logical order (split-major), so tiles reading the same pixel range
  // share that XCD's L2.
  if ((total & 7) == 0) {
    const int per = total >> 3;
    return (bid & 7) * per + (bid >> 3);
  }
  return bid;
}

template <int WM, int WN, int TM, int TN, int GM, int XG, bool RELU>
__global__ __launch_bounds__(WM * WN * 64, 8 / (WM * WN)) void k_wgrad_tr(WgTrK k) {
  constexpr int NT = WM * WN * 64;   // 4 or 8 waves
  constexpr int BN = WM * TM * 32, BK = WN * TN * 32;
  constexpr int GCH = BN / 8, XCH = BK / 8;   // 16-byte chunks per LDS row
  constexpr int GIT = (kMS * GCH + NT - 1) / NT, XIT = (kMS * XCH + NT - 1) / NT;
  __shared__ __attribute__((aligned(16))) bf16_t Gs[2][kMS * BN];
  __shared__ __attribute__((aligned(16))) bf16_t Xs[2][kMS * BK];

  const int tiles = k.tiles_n * k.tiles_k;
  const int bid = remap_block(blockIdx.x, gridDim.x);
  const int split = bid / tiles;
  const int tile = bid - split * tiles;
  const int tni = tile / k.tiles_k, tki = tile - tni * k.tiles_k;
  const int n0 = tni * BN, k0 = tki * BK;
  const int mbeg = split * k.m_per_split;
  const int mend = min(mbeg + k.m_per_split, k.M);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  // parity mode: class (pa, pb) of the gradient's pixels; the 2x2 filter's
  // tap (r, s) reads the source at (i + r - 1 + pa, j + s - 1 + pb)
  const int par = GM == kGParity ? (int)blockIdx.y : 0;
  const int pa = par >> 1, pb = par & 1;
  const int pad_r = GM == kGParity ? 1 - pa : k.pad, pad_s = GM == kGParity ? 1 - pb : k.pad;

  // ---- per-thread load slots (fixed across stages)
  int g_row[GIT], g_col[GIT], g_lds[GIT];
  bool g_on[GIT];
#pragma unroll
  for (int i = 0; i < GIT; ++i) {
    const int id = tid + NT * i;
    const int row = id / GCH, ch = id - (id / GCH) * GCH;
    g_on[i] = id < kMS * GCH && n0 + ch * 8 < k.Np;
    g_row[i] = row;
    g_col[i] = n0 + ch * 8;
    g_lds[i] = lds_off<BN>(row < kMS ? row : 0, ch * 8);
  }
  int x_row[XIT], x_rs[XIT], x_c[XIT], x_lds[XIT];
#pragma unroll
  for (int i = 0; i < XIT; ++i) {
    const int id = tid + NT * i;
    const int row = id / XCH, ch = id - (id / XCH) * XCH;
    const int kc = k0 + ch * 8;
    const bool on = id < kMS * XCH && kc < k.Kdim;
    const int tap = (int)fdiv((uint32_t)kc, k.fdC);
    const int c = kc - tap * k.C;
    const int r = (int)fdiv((uint32_t)tap, k.fdR);
    const int s = tap - r * k.R;
    x_row[i] = row;
    // tap offsets relative to the padding; an off slot gets an offset that
    // fails every bounds check
    x_rs[i] = on ? (((r - pad_r) & 0xffff) | ((s - pad_s) << 16)) : (0x4000 | (0x4000 << 16));
    x_c[i] = c;
    x_lds[i] = lds_off<BK>(row < kMS ? row : 0, ch * 8);
  }

  uint4 rg[GIT], rx[XIT];
  const __amdgpu_buffer_rsrc_t gr = make_rsrc(k.g, k.g_bytes);
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(k.x, k.x_bytes);
  auto load = [&](int mb) {
#pragma unroll
    for (int i = 0; i < GIT; ++i) {
      const int m = mb + g_row[i];
      int off;
      if (GM == kGDirect) {
        off = m * k.gC + g_col[i];
      } else {
        const int t = (int)fdiv((uint32_t)m, k.fdW);
        const int ow = m - t * k.W;
        const int b = (int)fdiv((uint32_t)t, k.fdH);
        const int oh = t - b * k.H;
        off = GM == kGUp2 ? ((b * k.Hs + (oh >> 1)) * k.Ws + (ow >> 1)) * k.gC + g_col[i]
                          : ((b * k.Hs + 2 * oh + pa) * k.Ws + 2 * ow + pb) * k.gC + g_col[i];
      }
      rg[i] = buf_ld16(gr, g_on[i] && m < mend ? 2u * (uint32_t)off : kOOB);
    }
#pragma unroll
    for (int i = 0; i < XIT; ++i) {
      const int m = mb + x_row[i];
      const int t = (int)fdiv((uint32_t)m, k.fdW);
      const int ow = m - t * k.W;
      const int b = (int)fdiv((uint32_t)t, k.fdH);
      const int oh = t - b * k.H;
      const int ih = (XG == G_S2 ? 2 * oh : oh) + (short)(x_rs[i] & 0xffff);
      const int iw = (XG == G_S2 ? 2 * ow : ow) + (x_rs[i] >> 16);
      const int hb = XG == G_S2 ? k.Hx : k.H, wb = XG == G_S2 ? k.Wx : k.W;
      const bool ok = m < mend && (unsigned)ih < (unsigned)hb && (unsigned)iw < (unsigned)wb;
      const int sh = XG == G_UP2 ? (ih >> 1) : ih, sw = XG == G_UP2 ? (iw >> 1) : iw;
      rx[i] = buf_ld16(xr, ok ? 2u * (uint32_t)(((b * k.Hx + sh) * k.Wx + sw) * k.C + x_c[i]) : kOOB);
    }
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int i = 0; i < GIT; ++i)
      if (tid + NT * i < kMS * GCH) *reinterpret_cast<uint4*>(&Gs[buf][g_lds[i]]) = rg[i];
#pragma unroll
    for (int i = 0; i < XIT; ++i)
      if (tid + NT * i < kMS * XCH)
        *reinterpret_cast<uint4*>(&Xs[buf][x_lds[i]]) = RELU ? relu8_bits(rx[i]) : rx[i];
  };

  // ---- per-lane transpose-read offsets: source lane L of a 16-lane group
  // addresses row 8*(L/32) + (L%16)/4 (+4 for the upper half of the K slice)
  // and column 16*((L/16)%2) + 4*(L%4) of its 32-column MFMA tile.
  const int rA = 8 * (lane >> 5) + ((lane & 15) >> 2);
  const int cA = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  int a_off[TM], b_off[TN];
#pragma unroll
  for (int i = 0; i < TM; ++i) a_off[i] = lds_off<BN>(rA, (wm * TM + i) * 32 + cA);
#pragma unroll
  for (int j = 0; j < TN; ++j) b_off[j] = lds_off<BK>(rA, (wn * TN + j) * 32 + cA);

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int nst = (mend - mbeg + kMS - 1) / kMS;
  if (nst > 0) {
    load(mbeg);
    store(0);
  }
  __syncthreads();
  int buf = 0;
  for (int st = 0; st < nst; ++st) {
    const bool more = st + 1 < nst;
    if (more) load(mbeg + (st + 1) * kMS);
    const bf16_t* gb = Gs[buf];
    const bf16_t* xb = Xs[buf];
    wg_step<TM, TN>(gb, xb, a_off, b_off, BN, BK, acc);
    if (more) store(buf ^ 1);
    __syncthreads();
    buf ^= 1;
  }

  float* part = k.part + ((int64_t)par * k.splits + split) * k.Np * k.Kdim;
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int kc = k0 + (wn * TN + j) * 32 + (lane & 31);
      if (kc >= k.Kdim) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int n = n0 + (wm * TM + i) * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        if (n < k.Np) part[(int64_t)n * k.Kdim + kc] = acc[i][j][r] * k.scale;
      }
    }
}


// ---- row-tap form of the direct 3x3 weight gradient
// For a 3x3, pad-1 conv over an image whose rows are multiples of 32 pixels
// wide, a 32-pixel stage lies in one image row, and the three taps (r, 0),
// (r, 1), (r, 2) of one filter row read that row's input at the 34 pixels
// ow0 - 1 .. ow0 + 32 shifted by 0, 1, 2.  A block here owns, for one filter
// row r and one 64-channel chunk, the 192 K columns (r, s, c0 .. c0 + 63),
// s = 0, 1, 2, and stages that 34 x 64 input segment once per 32 pixels: tap
// s's B operand is rows s .. s + 31 of it.  The activation bytes staged per
// MFMA drop to 34 / 96 of the tap-per-block form, whose operand loads bound
// it.  Gradient tile, transpose reads and fixed-order split reduction as in
// k_wgrad_tr.
template <int WM, int TM, int GM, bool RELU>
__global__ __launch_bounds__(WM * 2 * 64, 8 / (WM * 2)) void k_wgrad_row3(WgTrK k) {
  constexpr int WN = 2, TN = 3;
  constexpr int NT = WM * WN * 64;
  constexpr int BN = WM * TM * 32;
  constexpr int XR = 34, XC = 64;              // staged input rows (pixels) x channels
  constexpr int GCH = BN / 8;
  constexpr int GIT = (kMS * GCH + NT - 1) / NT, XIT = (XR * (XC / 8) + NT - 1) / NT;
  __shared__ __attribute__((aligned(16))) bf16_t Gs[2][kMS * BN];
  __shared__ __attribute__((aligned(16))) bf16_t Xs[2][36 * XC];

  const int cch = k.C / XC;                    // 64-channel chunks
  const int tiles = k.tiles_n * k.tiles_k;     // tiles_k = 3 filter rows x cch
  const int bid = remap_block(blockIdx.x, gridDim.x);
  const int split = bid / tiles;
  const int tile = bid - split * tiles;
  const int tni = tile / k.tiles_k, tki = tile - tni * k.tiles_k;
  const int fr = tki / cch, c0 = (tki - fr * cch) * XC;
  const int n0 = tni * BN;
  const int mbeg = split * k.m_per_split;
  const int mend = min(mbeg + k.m_per_split, k.M);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;

  int g_row[GIT], g_col[GIT], g_lds[GIT];
  bool g_on[GIT];
#pragma unroll
  for (int i = 0; i < GIT; ++i) {
    const int id = tid + NT * i;
    const int row = id / GCH, ch = id - (id / GCH) * GCH;
    g_on[i] = id < kMS * GCH && n0 + ch * 8 < k.Np;
    g_row[i] = row;
    g_col[i] = n0 + ch * 8;
    g_lds[i] = lds_off<BN>(row < kMS ? row : 0, ch * 8);
  }
  int x_row[XIT], x_ch[XIT], x_lds[XIT];
  bool x_on[XIT];
#pragma unroll
  for (int i = 0; i < XIT; ++i) {
    const int id = tid + NT * i;
    const int row = id / (XC / 8), ch = id - row * (XC / 8);
    x_on[i] = id < XR * (XC / 8);
    x_row[i] = row;
    x_ch[i] = ch;
    x_lds[i] = lds_off<XC>(x_on[i] ? row : 0, ch * 8);
  }

  uint4 rg[GIT], rx[XIT];
  const __amdgpu_buffer_rsrc_t gr = make_rsrc(k.g, k.g_bytes);
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(k.x, k.x_bytes);
  auto load = [&](int mb) {
#pragma unroll
    for (int i = 0; i < GIT; ++i) {
      const int m = mb + g_row[i];
      int off;
      if (GM == kGDirect) {
        off = m * k.gC + g_col[i];
      } else {
        const int t = (int)fdiv((uint32_t)m, k.fdW);
        const int ow = m - t * k.W;
        const int b = (int)fdiv((uint32_t)t, k.fdH);
        const int oh = t - b * k.H;
        off = ((b * k.Hs + (oh >> 1)) * k.Ws + (ow >> 1)) * k.gC + g_col[i];
      }
      rg[i] = buf_ld16(gr, g_on[i] && m < mend ? 2u * (uint32_t)off : kOOB);
    }
    // the stage's 32 pixels share one image row (b, oh), from column ow0
    const int t = (int)fdiv((uint32_t)mb, k.fdW);
    const int ow0 = mb - t * k.W;
    const int b = (int)fdiv((uint32_t)t, k.fdH);
    const int ih = t - b * k.H + fr - 1;
#pragma unroll
    for (int i = 0; i < XIT; ++i) {
      const int iw = ow0 - 1 + x_row[i];
      const bool ok = x_on[i] && (unsigned)ih < (unsigned)k.H && (unsigned)iw < (unsigned)k.W;
      rx[i] = buf_ld16(xr, ok ? 2u * (uint32_t)(((b * k.H + ih) * k.W + iw) * k.C + c0 + 8 * x_ch[i]) : kOOB);
    }
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int i = 0; i < GIT; ++i)
      if (tid + NT * i < kMS * GCH) *reinterpret_cast<uint4*>(&Gs[buf][g_lds[i]]) = rg[i];
#pragma unroll
    for (int i = 0; i < XIT; ++i)
      if (x_on[i]) *reinterpret_cast<uint4*>(&Xs[buf][x_lds[i]]) = RELU ? relu8_bits(rx[i]) : rx[i];
  };

  // transpose-read offsets as in k_wgrad_tr; B fragment j of this wave is
  // K columns 32 jj .. + 31 of the 192, jj = 3 wn + j: tap s = jj / 2,
  // channels 32 (jj % 2) .. of the chunk, read at rows shifted by s
  const int rA = 8 * (lane >> 5) + ((lane & 15) >> 2);
  const int cA = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  int a_off[TM], b_off[TN];
#pragma unroll
  for (int i = 0; i < TM; ++i) a_off[i] = lds_off<BN>(rA, (wm * TM + i) * 32 + cA);
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int jj = wn * TN + j;
    b_off[j] = lds_off<XC>(rA + (jj >> 1), 32 * (jj & 1) + cA);
  }

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int nst = (mend - mbeg + kMS - 1) / kMS;
  if (nst > 0) {
    load(mbeg);
    store(0);
  }
  __syncthreads();
  int buf = 0;
  for (int st = 0; st < nst; ++st) {
    const bool more = st + 1 < nst;
    if (more) load(mbeg + (st + 1) * kMS);
    const bf16_t* gb = Gs[buf];
    const bf16_t* xb = Xs[buf];
    wg_step<TM, TN>(gb, xb, a_off, b_off, BN, XC, acc);
    if (more) store(buf ^ 1);
    __syncthreads();
    buf ^= 1;
  }

  float* part = k.part + (int64_t)split * k.Np * k.Kdim;
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int jj = wn * TN + j;
    const int kc = (fr * 3 + (jj >> 1)) * k.C + c0 + 32 * (jj & 1) + (lane & 31);
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int n = n0 + (wm * TM + i) * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        if (n < k.Np) part[(int64_t)n * k.Kdim + kc] = acc[i][j][r] * k.scale;
      }
  }
}

// dw = scale * sum over splits, each output's splits added in split order.
// Up to 32 splits: a thread per 4 outputs (16-byte loads, four splits in
// flight); more: 256 outputs per block, 16 waves each summing every 16th
// split, then the 16 sums in wave order.  n is a multiple of 4 (Kdim is).
__global__ __launch_bounds__(256) void k_wgtr_reduce(const float* __restrict__ part, int splits, int64_t n4,
                                                     float scale, float* __restrict__ out) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n4) return;
  const float4* p = reinterpret_cast<const float4*>(part) + i;
  float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
  int j = 0;
  for (; j + 4 <= splits; j += 4) {
    float4 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = p[(int64_t)(j + u) * n4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      s.x += v[u].x; s.y += v[u].y; s.z += v[u].z; s.w += v[u].w;
    }
  }
  for (; j < splits; ++j) {
    const float4 v = p[(int64_t)j * n4];
    s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
  }
  reinterpret_cast<float4*>(out)[i] = make_float4(s.x * scale, s.y * scale, s.z * scale, s.w * scale);
}

__global__ __launch_bounds__(1024) void k_wgtr_reduce_wide(const float* __restrict__ part, int splits, int64_t n4,
                                                           float scale, float* __restrict__ out) {
  __shared__ float4 sh[16][64];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int64_t i = (int64_t)blockIdx.x * 64 + lane;
  const float4* p = reinterpret_cast<const float4*>(part) + i;
  float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
  if (i < n4)
    for (int j = wv; j < splits; j += 16) {
      const float4 v = p[(int64_t)j * n4];
      s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
    }
  sh[wv][lane] = s;
  __syncthreads();
  if (wv == 0 && i < n4) {
    float4 t = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int w = 0; w < 16; ++w) {
      t.x += sh[w][lane].x; t.y += sh[w][lane].y; t.z += sh[w][lane].z; t.w += sh[w][lane].w;
    }
    reinterpret_cast<float4*>(out)[i] = make_float4(t.x * scale, t.y * scale, t.z * scale, t.w * scale);
  }
}

// Fold of the sub-pixel weight gradients onto the 3x3 filter:
//   dw[n][r][s][c] = scale * sum over parities (a, b), then splits, of
//                    part[(2a + b) * splits + sp][n][(D_a(r) * 2 + D_b(s)) * C + c],
// D_0 = (0, 1, 1), D_1 = (0, 0, 1): the 2x2 tap that 3x3 tap r feeds in
// parity class a.  Four consecutive channels per thread (C % 4 == 0).
__global__ __launch_bounds__(256) void k_wgrad_fold_sub(const float* __restrict__ part, int splits, int Np, int C,
                                                        float scale, float* __restrict__ dw) {
  const int C4 = C / 4;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (int64_t)Np * 9 * C4) return;
  const int c4 = (int)(i % C4);
  const int64_t t = i / C4;
  const int tap = (int)(t % 9), n = (int)(t / 9);
  const int r = tap / 3, s_ = tap % 3;
  const int64_t plane = (int64_t)Np * 4 * C;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
  for (int ab = 0; ab < 4; ++ab) {
    const int a = ab >> 1, b = ab & 1;
    const int du = a == 0 ? (r > 0) : (r == 2), dv = b == 0 ? (s_ > 0) : (s_ == 2);
    const float* src = part + (int64_t)ab * splits * plane + ((int64_t)n * 4 + du * 2 + dv) * C + 4 * c4;
    for (int sp = 0; sp < splits; ++sp) {
      const float4 v = *reinterpret_cast<const float4*>(src + sp * plane);
      acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
    }
  }
  reinterpret_cast<float4*>(dw)[i] = make_float4(acc.x * scale, acc.y * scale, acc.z * scale, acc.w * scale);
}

struct TrCfg {
  int WM, WN, TM, TN;
};
constexpr TrCfg kTrCfgs[] = {{2, 2, 4, 2}, {2, 2, 2, 4}, {2, 2, 3, 3}, {1, 4, 3, 2}, {1, 4, 3, 3}, {2, 2, 2, 2},
                             {4, 2, 2, 4}};
constexpr int kTrWide = 6;   // the eight-wave 256 x 256 tile

struct TrPlan {
  int cfg, tiles_n, tiles_k, splits, m_per_split;
};

// Tile shape with the least padded work (BigGAN widths are multiples of 96,
// filter-tap K dims multiples of 288), then a split of the pixel range that
// gives the chip ~4 blocks per CU, each split at least 1024 pixels long.
TrPlan tr_plan(int64_t M, int R, int Cin, int Np, int n_cu) {
  const int64_t K = (int64_t)R * R * Cin;
  TrPlan p{0, 0, 0, 1, 0};
  double best = 1e300;
  for (int c = 0; c < (int)(sizeof(kTrCfgs) / sizeof(kTrCfgs[0])); ++c) {
    const TrCfg& t = kTrCfgs[c];
    const int bn = t.WM * t.TM * 32, bk = t.WN * t.TN * 32;
    const double tiles = (double)cdiv(Np, bn) * cdiv(K, bk);
    const double eff = t.TM * t.TN >= 8 ? 1.0 : (t.TM * t.TN >= 6 ? 0.92 : 0.8);
    const double cost = tiles * bn * bk / eff;
    if (cost < best * 0.999) {
      best = cost;
      p.cfg = c;
    }
  }
  // 256 x 256 on eight waves (one block per CU) where both dimensions are
  // multiples of 256: half the operand bytes per MFMA of 256 x 128
  // (measured 5-13 % faster on the 768 / 1536-channel weight gradients)
  if (Np % 256 == 0 && K % 256 == 0) p.cfg = kTrWide;
  const TrCfg& t = kTrCfgs[p.cfg];
  p.tiles_n = (int)cdiv(Np, t.WM * t.TM * 32);
  p.tiles_k = (int)cdiv(K, t.WN * t.TN * 32);
  const int64_t tiles = (int64_t)p.tiles_n * p.tiles_k;
  const int64_t smax = std::max<int64_t>(1, M / 1024);
  const int64_t cap = (512LL << 20) / (4 * (int64_t)Np * K);
  int64_t sp;
  if (p.cfg == kTrWide) {
    // ~1 block per CU (each split's partial sums cost a write and a read in
    // the reduction), then the split count up to twice that whose blocks
    // fill the last round over the CUs best
    const int64_t s0 = std::max<int64_t>(1, std::min({cdiv((int64_t)n_cu, tiles), smax, cap}));
    sp = s0;
    double best_fill = 0.0;
    for (int64_t c = s0; c <= std::min({2 * s0, smax, cap}); ++c) {
      const int64_t b = c * tiles;
      const double fill = (double)b / (double)(cdiv(b, (int64_t)n_cu) * n_cu);
      if (fill > best_fill + 1e-9) {
        best_fill = fill;
        sp = c;
      }
    }
  } else {
    sp = cdiv(4LL * n_cu, tiles);
    sp = std::min<int64_t>(sp, smax);
    sp = std::max<int64_t>(1, std::min<int64_t>(sp, cap));
  }
  p.m_per_split = (int)(cdiv(cdiv(M, sp), kMS) * kMS);
  p.splits = (int)cdiv(M, p.m_per_split);
  return p;
}

template <int WM, int WN, int TM, int TN>
std::string launch_tr(hipStream_t s, const WgTrK& k, int blocks, int gm, int xg, bool relu) {
#define PG_WTR_CASE(GM, XG, RL, NAME)                                                                      \
  if (gm == GM && xg == XG && relu == RL) {                                                                \
    hipLaunchKernelGGL((k_wgrad_tr<WM, WN, TM, TN, GM, XG, RL>), dim3(blocks, GM == kGParity ? 4 : 1),      \
                       dim3(64 * WM * WN), 0, s, k);                                                       \
    return "k_wgrad_tr<" + std::to_string(WM * TM * 32) + "x" + std::to_string(WN * TN * 32) + "," NAME "," \
           #XG "," #RL ">";                                                                                \
  }
  PG_WTR_CASE(kGDirect, G_DIRECT, false, "false")
  PG_WTR_CASE(kGDirect, G_DIRECT, true, "false")
  PG_WTR_CASE(kGUp2, G_DIRECT, false, "true")
  PG_WTR_CASE(kGUp2, G_DIRECT, true, "true")
  PG_WTR_CASE(kGDirect, G_UP2, false, "false")
  PG_WTR_CASE(kGDirect, G_S2, true, "false")
  PG_WTR_CASE(kGParity, G_DIRECT, false, "SUB")
#undef PG_WTR_CASE
  throw Error{-2, "wgrad_tr: unsupported gather combination"};
}

// the row-tap kernel: 192 or 256 output channels per block
template <int WM, int TM>
std::string launch_row3(hipStream_t s, const WgTrK& k, int blocks, int gm, bool relu) {
#define PG_ROW3_CASE(GM, RL, GNAME)                                                                    \
  if (gm == GM && relu == RL) {                                                                        \
    hipLaunchKernelGGL((k_wgrad_row3<WM, TM, GM, RL>), dim3(blocks), dim3(64 * WM * 2), 0, s, k);     \
    return "k_wgrad_row3<" + std::to_string(WM * TM * 32) + "x192," GNAME "," #RL ">";                \
  }
  PG_ROW3_CASE(kGDirect, false, "false")
  PG_ROW3_CASE(kGDirect, true, "false")
  PG_ROW3_CASE(kGUp2, false, "true")
  PG_ROW3_CASE(kGUp2, true, "true")
#undef PG_ROW3_CASE
  throw Error{-2, "wgrad_row3: unsupported gradient gather"};
}

std::string launch_cfg_tr(hipStream_t s, int cfg, const WgTrK& k, int blocks, int gm, int xg, bool relu) {
  switch (cfg) {
    case 0: return launch_tr<2, 2, 4, 2>(s, k, blocks, gm, xg, relu);
    case 1: return launch_tr<2, 2, 2, 4>(s, k, blocks, gm, xg, relu);
    case 2: return launch_tr<2, 2, 3, 3>(s, k, blocks, gm, xg, relu);
    case 3: return launch_tr<1, 4, 3, 2>(s, k, blocks, gm, xg, relu);
    case 4: return launch_tr<1, 4, 3, 3>(s, k, blocks, gm, xg, relu);
    case 5: return launch_tr<2, 2, 2, 2>(s, k, blocks, gm, xg, relu);
    default: return launch_tr<4, 2, 2, 4>(s, k, blocks, gm, xg, relu);
  }
}

}  // namespace

bool wgrad_tr_ok(const GradIn& g, const ConvIn& in, int H, int W, int R, int Np) {
  if (in.mean || in.gather == G_POOL2 || in.gscale != 1.f) return false;
  if (in.gather == G_UP2 && in.relu) return false;
  if (in.gather == G_S2 && (R != 4 || in.Hx != 2 * H || in.Wx != 2 * W || g.gather != G_DIRECT)) return false;
  if (g.gather != G_DIRECT && g.gather != G_UP2) return false;
  const int64_t M = (int64_t)in.B * H * W;
  const int64_t xs = (int64_t)in.B * in.Hx * in.Wx * in.C;
  const int64_t gs = g.gather == G_DIRECT ? M * g.C : (int64_t)in.B * g.Hs * g.Ws * g.C;
  return M < (1LL << 30) && xs < (1LL << 31) && gs < (1LL << 31) && 2 * xs < kBufMax && 2 * gs < kBufMax &&
         in.C % 8 == 0 && g.C % 8 == 0 && Np % 8 == 0;
}

size_t wgrad_tr_ws(int64_t M, int R, int Cin, int Np, int n_cu) {
  const TrPlan p = tr_plan(M, R, Cin, Np, n_cu);
  return p.splits > 1 ? align256((size_t)p.splits * Np * R * R * Cin * 4) : 0;
}

void wgrad_tr(hipStream_t s, const GradIn& g, const ConvIn& in, int H, int W, int R, int Np, float* dw,
              void* ws, size_t ws_bytes, int n_cu, double flops) {
  WgTrK k;
  k.g = (const bf16_t*)g.g;
  k.x = (const bf16_t*)in.x;
  k.x_bytes = 2LL * in.B * in.Hx * in.Wx * in.C;
  k.g_bytes = 2LL * (g.gather == G_DIRECT ? (int64_t)in.B * H * W : (int64_t)in.B * g.Hs * g.Ws) * g.C;
  k.gC = g.C;
  k.Np = Np;
  k.Kdim = R * R * in.C;
  k.C = in.C;
  k.R = R;
  k.pad = in.gather == G_S2 ? 1 : R / 2;
  k.H = H;
  k.W = W;
  k.Hx = in.Hx;
  k.Wx = in.Wx;
  k.Hs = g.Hs;
  k.Ws = g.Ws;
  k.M = (int)((int64_t)in.B * H * W);
  k.fdW = make_fastdiv(W);
  k.fdH = make_fastdiv(H);
  k.fdC = make_fastdiv(in.C);
  k.fdR = make_fastdiv(R);
  const TrPlan p = tr_plan(k.M, R, in.C, Np, n_cu);
  k.m_per_split = p.m_per_split;
  k.tiles_n = p.tiles_n;
  k.tiles_k = p.tiles_k;
  k.splits = p.splits;
  // the row-tap form (k_wgrad_row3): a direct 3x3 conv over images whose
  // rows are whole 32-pixel stages, 64-channel chunks, 192 / 256-channel
  // output tiles; same splits (so the same partial buffer)
  const bool row3 = R == 3 && in.gather == G_DIRECT && W % 32 == 0 && in.C % 64 == 0 &&
                    (Np % 256 == 0 || Np % 192 == 0) && k.M % 32 == 0;
  if (row3) {
    k.tiles_n = Np / (Np % 256 == 0 ? 256 : 192);
    k.tiles_k = 3 * (in.C / 64);
  }
  const int64_t nout = (int64_t)Np * k.Kdim;
  if (p.splits > 1 && (size_t)p.splits * nout * 4 > ws_bytes) throw Error{-3, "conv_wgrad: workspace too small"};
  PG_CHECK(p.splits == 1 || (nout % 4 == 0 && (((uintptr_t)ws | (uintptr_t)dw) & 15) == 0),
           "conv_wgrad: split partials must be 16-byte aligned rows of whole float4s");
  // a single split writes the scaled result itself; several leave unscaled partials
  k.part = p.splits == 1 ? dw : (float*)ws;
  k.scale = p.splits == 1 ? g.gscale : 1.f;
  const int blocks = p.splits * k.tiles_n * k.tiles_k;
  const int gm = g.gather == G_UP2 ? kGUp2 : kGDirect;
  std::string name;
  ProfScope prof(s);
  if (row3)
    name = Np % 256 == 0 ? launch_row3<4, 2>(s, k, blocks, gm, in.relu) : launch_row3<2, 3>(s, k, blocks, gm, in.relu);
  else
    name = launch_cfg_tr(s, p.cfg, k, blocks, gm, in.gather, in.relu);
  PG_LAUNCH_CHECK();
  prof.done(name, flops, k.M, Np, k.Kdim);
  if (p.splits > 1) {
    ProfScope pr(s);
    const int64_t n4 = nout / 4;
    if (p.splits <= 32)
      hipLaunchKernelGGL(k_wgtr_reduce, dim3((unsigned)cdiv(n4, 256)), dim3(256), 0, s, k.part, p.splits, n4,
                         g.gscale, dw);
    else
      hipLaunchKernelGGL(k_wgtr_reduce_wide, dim3((unsigned)cdiv(n4, 64)), dim3(1024), 0, s, k.part, p.splits, n4,
                         g.gscale, dw);
    PG_LAUNCH_CHECK();
    pr.done("k_wgtr_reduce", 0.0);
  }
}

// ---- sub-pixel weight gradient of a 3x3 conv over a nearest 2x upsample
// The forward runs that conv as four 2x2 convs over the source grid, one per
// parity class (a, b) of the output pixels, each with the filter sums
//   W_ab[n][du][dv] = sum of W[n][r][s] over r in S(a, du), s in S(b, dv)
// (S(a, 0) = [0, a], S(a, 1) = [1 + a, 2]).  Each 3x3 tap sits in exactly one
// sum per class, so dW[n][r][s] = sum over (a, b) of dW_ab[n][D_a(r)][D_b(s)],
// and dW_ab = sum over the class's pixels of dY (x) (the 2x2 window of the
// source): 4/9 of the upsampled form's MACs, on the unexpanded source.
static TrPlan sub_plan(int64_t Msrc, int Cin, int Np, int n_cu) {
  // four parity classes share the CUs
  return tr_plan(Msrc, 2, Cin, Np, std::max(1, n_cu / 4));
}

size_t wgrad_sub_ws(int64_t Msrc, int Cin, int Np, int n_cu) {
  const TrPlan p = sub_plan(Msrc, Cin, Np, n_cu);
  return align256((size_t)4 * p.splits * Np * 4 * Cin * 4);
}

bool wgrad_sub_ok(const GradIn& g, const ConvIn& in, int Np) {
  if (in.mean || in.relu || in.gather != G_DIRECT || g.gather != G_DIRECT || in.gscale != 1.f) return false;
  const int64_t xs = (int64_t)in.B * in.Hx * in.Wx * in.C;
  const int64_t gs = (int64_t)in.B * g.Hs * g.Ws * g.C;
  return g.Hs == 2 * in.Hx && g.Ws == 2 * in.Wx && xs < (1LL << 31) && gs < (1LL << 31) && 2 * xs < kBufMax &&
         2 * gs < kBufMax && in.C % 8 == 0 && g.C % 8 == 0 && Np % 8 == 0;
}

void wgrad_sub(hipStream_t s, const GradIn& g, const ConvIn& in, int Np, float* dw, void* ws, size_t ws_bytes,
               int n_cu) {
  PG_CHECK(wgrad_sub_ok(g, in, Np), "wgrad_sub: operands");
  const int H = in.Hx, W = in.Wx;
  WgTrK k;
  k.g = (const bf16_t*)g.g;
  k.x = (const bf16_t*)in.x;
  k.x_bytes = 2LL * in.B * H * W * in.C;
  k.g_bytes = 2LL * in.B * g.Hs * g.Ws * g.C;
  k.gC = g.C;
  k.Np = Np;
  k.Kdim = 4 * in.C;
  k.C = in.C;
  k.R = 2;
  k.pad = 0;   // per parity in the kernel
  k.H = H;
  k.W = W;
  k.Hx = H;
  k.Wx = W;
  k.Hs = g.Hs;
  k.Ws = g.Ws;
  k.M = (int)((int64_t)in.B * H * W);
  k.fdW = make_fastdiv(W);
  k.fdH = make_fastdiv(H);
  k.fdC = make_fastdiv(in.C);
  k.fdR = make_fastdiv(2);
  const TrPlan p = sub_plan(k.M, in.C, Np, n_cu);
  k.m_per_split = p.m_per_split;
  k.tiles_n = p.tiles_n;
  k.tiles_k = p.tiles_k;
  k.splits = p.splits;
  const size_t need = (size_t)4 * p.splits * Np * k.Kdim * 4;
  if (need > ws_bytes) throw Error{-3, "wgrad_sub: workspace too small"};
  PG_CHECK(in.C % 4 == 0 && (((uintptr_t)ws | (uintptr_t)dw) & 15) == 0, "wgrad_sub: alignment");
  k.part = (float*)ws;
  k.scale = 1.f;
  const int blocks = p.splits * p.tiles_n * p.tiles_k;
  ProfScope prof(s);
  const std::string name = launch_cfg_tr(s, p.cfg, k, blocks, kGParity, G_DIRECT, false);
  PG_LAUNCH_CHECK();
  // executed MACs: four classes of M source pixels x 4 taps
  const double flops = 2.0 * 4.0 * k.M * (g.n_real ? g.n_real : Np) * 4.0 * (in.c_real ? in.c_real : in.C);
  prof.done(name, flops, 4LL * k.M, Np, k.Kdim);
  ProfScope pr(s);
  const int64_t n4 = (int64_t)Np * 9 * in.C / 4;
  hipLaunchKernelGGL(k_wgrad_fold_sub, dim3((unsigned)cdiv(n4, 256)), dim3(256), 0, s, (const float*)k.part,
                     p.splits, Np, in.C, g.gscale, dw);
  PG_LAUNCH_CHECK();
  pr.done("k_wgrad_fold_sub", 0.0);
}

}  // namespace pg
