// Self-attention core on gfx950 (bf16 MFMA 32x32x16, fp32 softmax).
//
// Per image: queries theta (HW x dk), keys phi and values g max-pooled 2x2
// (L = HW/4 rows), scores S = Q K^T without scaling, softmax over keys,
// O = P V.  Flash-style: S is never stored.  The scores are computed
// transposed (S^T = K Q^T), so each lane owns one query (forward, dQ) or one
// key (dK, dV) and the softmax reductions stay in-lane plus one swap with the
// lane 32 apart.  Probabilities feed the next product straight from the
// accumulator registers: the 8 k-slots of lane group g (lane / 32) hold the
// rows {4g..4g+3, 8+4g..8+4g+3} (+16 per k-step) of the score tile, and the
// other operand is read in that same row order.
//
// The operand that every wave of a block shares (a 32-row block of keys and
// values, or of queries and output gradients) is staged in LDS once per
// block; row-major MFMA operands come out of it with 16-byte reads and the
// transposed ones (V^T, K^T, Q^T, dO^T) with ds_read_b64_tr_b16, so no
// transposed copy exists in memory.  LDS rows are swizzled in 16-byte chunks
// so that both kinds of read are free of bank conflicts.
//
// Exponentials are base 2: the saved log-sum-exp is in log2 units and the
// running maximum of the forward is only raised when the block maximum
// exceeds it by more than 2^8 (the rescale of the accumulators is then rare;
// unnormalised probabilities stay below 2^8).
//
// Layouts (bf16 unless noted), per image b, key count padded to Lp = 32k
// and query count to HWp = 32k:
//   qkv [HW][Nqkv]   projections, theta | phi | g at channel offsets 0, dk, 2dk
//   kp [Lp][dk], vp [Lp][dv]   pooled keys / values, rows >= L zero
//   o, dO [HW][dv];  lse2, Dv [HWp] fp32 (lse2 = +inf for padded queries)
#include "attn.hpp"

namespace pg {

namespace {

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
constexpr float kL2E = 1.4426950408889634f;   // log2(e)
constexpr float kTau = 8.f;                   // lazy-rescale threshold (log2 units)

PG_DEV bf16x8 ld8g(const bf16_t* p) { return *reinterpret_cast<const bf16x8*>(p); }
PG_DEV bf16x8 zero8() {
  uint4 q = make_uint4(0, 0, 0, 0);
  return *reinterpret_cast<bf16x8*>(&q);
}
PG_DEV bf16x8 pack_regs(const f32x16& v, int t) {
  const uint4 q = make_uint4(f2bf2(v[8 * t], v[8 * t + 1]), f2bf2(v[8 * t + 2], v[8 * t + 3]),
                             f2bf2(v[8 * t + 4], v[8 * t + 5]), f2bf2(v[8 * t + 6], v[8 * t + 7]));
  return __builtin_bit_cast(bf16x8, q);
}
// row index (within a 32-tile) held by accumulator register r of lane group g
PG_DEV int acc_row(int r, int g) { return 8 * (r >> 2) + 4 * g + (r & 3); }
PG_DEV float exp2_(float x) { return __builtin_amdgcn_exp2f(x); }

// ---- LDS tiles: rows of NC 16-byte chunks, chunk index XOR-swizzled by row
template <int NC>
PG_DEV int swz16(int r) {
  if (NC == 8) return ((r >> 2) & 3) | (((r >> 1) & 1) << 2);
  if (NC == 16) return 4 * (r & 3) + ((r >> 2) & 3);
  return (r >> 2) & 3;   // NC = 4 or 12
}
template <int NC>
PG_DEV int toff(int r, int e) {
  return r * NC * 8 + ((((e >> 3) ^ swz16<NC>(r))) << 3) + (e & 7);
}
// row-major operand: 8 consecutive elements of row r starting at e (e % 8 == 0)
template <int NC>
PG_DEV bf16x8 ld_row(const bf16_t* t, int r, int e) {
  return *reinterpret_cast<const bf16x8*>(t + toff<NC>(r, e));
}
// transposed operand: column c0 + lane%32 of rows {16kk + 4g + 0..3, 16kk + 8 + 4g + 0..3}
template <int NC>
PG_DEV bf16x8 ld_tr(const bf16_t* t, int kk, int c0, int lane) {
  const int r = 16 * kk + 4 * (lane >> 5) + ((lane & 15) >> 2);
  const int c = c0 + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(t + toff<NC>(r, c)));
  const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(t + toff<NC>(r + 8, c)));
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

// Stage rows [r0, r0 + 32) x NC chunks of a row-major source (row stride ld
// elements) into a swizzled tile; rows >= nrows are zero.  Thread slots
// i = tid + 256 j.
template <int NC, int SLOTS>
struct Stager {
  uint4 v[SLOTS];
  PG_DEV void load(const bf16_t* src, int64_t ld, int r0, int nrows, int tid) {
#pragma unroll
    for (int j = 0; j < SLOTS; ++j) {
      const int i = tid + 256 * j;
      const int r = i / NC, c = i - (i / NC) * NC;
      v[j] = make_uint4(0, 0, 0, 0);
      if (i < 32 * NC && r0 + r < nrows) v[j] = *reinterpret_cast<const uint4*>(src + (int64_t)(r0 + r) * ld + c * 8);
    }
  }
  PG_DEV void store(bf16_t* t, int tid) const {
#pragma unroll
    for (int j = 0; j < SLOTS; ++j) {
      const int i = tid + 256 * j;
      const int r = i / NC, c = i - (i / NC) * NC;
      if (i < 32 * NC) *reinterpret_cast<uint4*>(t + toff<NC>(r, c * 8)) = v[j];
    }
  }
};

}  // namespace

// ------------------------------------------------------------- pooling
// Max over each 2x2 window (first maximum in (dh, dw) row-major order wins)
// of the phi and g channels; writes K and V, rows >= L zero.
// 2x2 max pool of the key / value projections, 8 channels per thread
// (16-byte loads and stores); ties keep the first of the window in row
// order; rows l >= L of the padded outputs are zero.
__global__ void k_attn_pool(const bf16_t* qkv, int B, int H, int W, int Nqkv, int dk, int dv, int Lp, bf16_t* kp,
                            bf16_t* vp) {
  const int L = (H / 2) * (W / 2);
  const int ng = (dk + dv) / 8;
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= B * Lp * ng) return;
  const int g = i % ng, t = i / ng;
  const int l = t % Lp, b = t / Lp;
  const int c = 8 * g;
  uint4 best = make_uint4(0u, 0u, 0u, 0u);
  if (l < L) {
    const int ph = l / (W / 2), pw = l - ph * (W / 2);
    float bv[8];
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      const int h = 2 * ph + (d >> 1), w = 2 * pw + (d & 1);
      const uint4 q = *reinterpret_cast<const uint4*>(qkv + ((int64_t)(b * H + h) * W + w) * Nqkv + dk + c);
      float v[8];
      unpack8(q, v);
      uint32_t* bw = reinterpret_cast<uint32_t*>(&best);
      const uint32_t* qw = reinterpret_cast<const uint32_t*>(&q);
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (d == 0 || v[e] > bv[e]) {
          bv[e] = v[e];
          const uint32_t half = (qw[e >> 1] >> (16 * (e & 1))) & 0xffffu;
          bw[e >> 1] = (bw[e >> 1] & ~(0xffffu << (16 * (e & 1)))) | (half << (16 * (e & 1)));
        }
    }
  }
  if (c < dk)
    *reinterpret_cast<uint4*>(kp + ((int64_t)b * Lp + l) * dk + c) = best;
  else
    *reinterpret_cast<uint4*>(vp + ((int64_t)b * Lp + l) * dv + c - dk) = best;
}

// ------------------------------------------------------------- forward
// A wave owns 2 query tiles (64 queries); a block of 4 waves 256 queries.
template <int DV>
__global__ __launch_bounds__(256, 2) void k_attn_fwd(const bf16_t* qkv, int Nqkv, const bf16_t* kp,
                                                     const bf16_t* vp, int HW, int L, int Lp, int HWp, bf16_t* o,
                                                     float* o32, float* lse2) {
  constexpr int DK = 32, NT = DV / 32, NCV = DV / 8, QT = 2;
  __shared__ __attribute__((aligned(16))) bf16_t Ks[2][32 * DK];
  __shared__ __attribute__((aligned(16))) bf16_t Vs[2][32 * DV];
  const int b = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 5, lq = lane & 31;
  const int qw = blockIdx.x * 256 + (tid >> 6) * 64;
  const bf16_t* Q = qkv + (int64_t)b * HW * Nqkv;
  const bf16_t* K = kp + (int64_t)b * Lp * DK;
  const bf16_t* V = vp + (int64_t)b * Lp * DV;
  bf16x8 qb[QT][2];
#pragma unroll
  for (int u = 0; u < QT; ++u) {
    const int q = qw + 32 * u + lq;
#pragma unroll
    for (int t = 0; t < 2; ++t) qb[u][t] = q < HW ? ld8g(Q + (int64_t)q * Nqkv + 16 * t + 8 * g) : zero8();
  }
  f32x16 acc[QT][NT];
#pragma unroll
  for (int u = 0; u < QT; ++u)
#pragma unroll
    for (int j = 0; j < NT; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[u][j][r] = 0.f;
  float m2[QT], l[QT];
#pragma unroll
  for (int u = 0; u < QT; ++u) { m2[u] = -INFINITY; l[u] = 0.f; }

  Stager<4, 1> sk;
  Stager<NCV, (32 * NCV + 255) / 256> sv;
  sk.load(K, DK, 0, Lp, tid);
  sv.load(V, DV, 0, Lp, tid);
  sk.store(Ks[0], tid);
  sv.store(Vs[0], tid);
  __syncthreads();
  int buf = 0;
  for (int k0 = 0; k0 < Lp; k0 += 32) {
    const bool more = k0 + 32 < Lp;
    if (more) {
      sk.load(K, DK, k0 + 32, Lp, tid);
      sv.load(V, DV, k0 + 32, Lp, tid);
    }
    const bf16_t* ks = Ks[buf];
    const bf16_t* vs = Vs[buf];
    f32x16 s[QT];
#pragma unroll
    for (int u = 0; u < QT; ++u)
#pragma unroll
      for (int r = 0; r < 16; ++r) s[u][r] = 0.f;
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const bf16x8 ka = ld_row<4>(ks, lq, 16 * t + 8 * g);
#pragma unroll
      for (int u = 0; u < QT; ++u) s[u] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qb[u][t], s[u], 0, 0, 0);
    }
    const bool tail = k0 + 32 > L;
#pragma unroll
    for (int u = 0; u < QT; ++u) {
      if (tail) {
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (k0 + acc_row(r, g) >= L) s[u][r] = -INFINITY;
      }
      float mb = s[u][0];
#pragma unroll
      for (int r = 1; r < 16; ++r) mb = fmaxf(mb, s[u][r]);
      mb = fmaxf(mb, __shfl_xor(mb, 32, 64)) * kL2E;
      if (mb > m2[u] + kTau) {
        const float alpha = exp2_(m2[u] - mb);
        l[u] *= alpha;
#pragma unroll
        for (int j = 0; j < NT; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[u][j][r] *= alpha;
        m2[u] = mb;
      }
      float ls = 0.f;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        s[u][r] = exp2_(fmaf(s[u][r], kL2E, -m2[u]));
        ls += s[u][r];
      }
      l[u] += ls;
    }
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      bf16x8 pb[QT];
#pragma unroll
      for (int u = 0; u < QT; ++u) pb[u] = pack_regs(s[u], t);
#pragma unroll
      for (int j = 0; j < NT; ++j) {
        const bf16x8 va = ld_tr<NCV>(vs, t, 32 * j, lane);
#pragma unroll
        for (int u = 0; u < QT; ++u) acc[u][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb[u], acc[u][j], 0, 0, 0);
      }
    }
    if (more) {
      sk.store(Ks[buf ^ 1], tid);
      sv.store(Vs[buf ^ 1], tid);
    }
    __syncthreads();
    buf ^= 1;
  }
#pragma unroll
  for (int u = 0; u < QT; ++u) {
    const int q = qw + 32 * u + lq;
    const float lt = l[u] + __shfl_xor(l[u], 32, 64);
    const float inv = 1.f / lt;
    // fp32 copy in register layout: 32-query tile, then (j, i), then lane:
    // every store is 64 lanes x 16 contiguous bytes
    float4* const t32 = o32 && qw + 32 * u < HWp
                            ? reinterpret_cast<float4*>(o32 + ((int64_t)b * (HWp / 32) + (qw + 32 * u) / 32) * DV * 32)
                            : nullptr;
    bf16_t* orow = o + ((int64_t)b * HW + q) * DV;
#pragma unroll
    for (int j = 0; j < NT; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const f32x16& a = acc[u][j];
        const float4 f = make_float4(a[4 * i] * inv, a[4 * i + 1] * inv, a[4 * i + 2] * inv, a[4 * i + 3] * inv);
        if (q < HW) *reinterpret_cast<uint2*>(orow + 32 * j + 8 * i + 4 * g) = make_uint2(f2bf2(f.x, f.y), f2bf2(f.z, f.w));
        if (t32) t32[(j * 4 + i) * 64 + lane] = f;
      }
    if (g == 0 && q < HWp) lse2[(int64_t)b * HWp + q] = q < HW ? m2[u] + __log2f(lt) : INFINITY;
  }
}

// ------------------------------------------------------------- dQ (query-owned)
// One pass over the keys: dS = P (dP - Dv) and dQ^T = K^T dS^T, where the
// softmax backward's row term Dv[q] = sum_k P dP = dO[q] . O[q] is the dot
// product of the query's output gradient with the forward's fp32 output row
// (normalised accumulators, before bf16 rounding), formed in the prologue.
template <int DV>
constexpr int dq_tiles() { return DV >= 96 ? 1 : 2; }   // query tiles per wave (register budget)

template <int DV>
__global__ __launch_bounds__(256, 2) void k_attn_dq(const bf16_t* qkv, int Nqkv, const bf16_t* kp,
                                                    const bf16_t* vp, const bf16_t* dO, const float* O32,
                                                    const float* lse2, float* Dv, int HW, int L, int Lp, int HWp,
                                                    bf16_t* dqkv) {
  constexpr int DK = 32, NCV = DV / 8, QT = dq_tiles<DV>();
  __shared__ __attribute__((aligned(16))) bf16_t Ks[2][32 * DK];
  __shared__ __attribute__((aligned(16))) bf16_t Vs[2][32 * DV];
  const int b = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 5, lq = lane & 31;
  const int qw = blockIdx.x * 128 * QT + (tid >> 6) * 32 * QT;
  const bf16_t* Q = qkv + (int64_t)b * HW * Nqkv;
  const bf16_t* K = kp + (int64_t)b * Lp * DK;
  const bf16_t* V = vp + (int64_t)b * Lp * DV;
  const bf16_t* DO = dO + (int64_t)b * HW * DV;
  const float4* OO = reinterpret_cast<const float4*>(O32 + (int64_t)b * HWp * DV);
  bf16x8 qb[QT][2], db[QT][DV / 16];
  float lq2[QT], dd[QT];
  bool qv[QT];
#pragma unroll
  for (int u = 0; u < QT; ++u) {
    const int q = qw + 32 * u + lq;
    qv[u] = q < HW;
#pragma unroll
    for (int t = 0; t < 2; ++t) qb[u][t] = qv[u] ? ld8g(Q + (int64_t)q * Nqkv + 16 * t + 8 * g) : zero8();
    dd[u] = 0.f;
#pragma unroll
    for (int t = 0; t < DV / 16; ++t) {
      db[u][t] = qv[u] ? ld8g(DO + (int64_t)q * DV + 16 * t + 8 * g) : zero8();
      // this lane's half of dO[q] . O[q] (channels 16 t + 8 g ..)
      if (qv[u]) {
        // channels 16 t + 8 g + 0..7 of query q: in the forward's register
        // layout (j, i) = (t / 2, 2 (t % 2) + g), lanes lq and 32 + lq
        float a[8];
        unpack8(__builtin_bit_cast(uint4, db[u][t]), a);
        const float4* tile = OO + (int64_t)((qw + 32 * u) / 32) * DV * 8;
        const int ji = (t / 2) * 4 + 2 * (t % 2) + g;
        const float4 o0 = tile[ji * 64 + lq], o1 = tile[ji * 64 + 32 + lq];
        const float o[8] = {o0.x, o0.y, o0.z, o0.w, o1.x, o1.y, o1.z, o1.w};
#pragma unroll
        for (int e = 0; e < 8; ++e) dd[u] = fmaf(a[e], o[e], dd[u]);
      }
    }
    lq2[u] = qv[u] ? lse2[(int64_t)b * HWp + q] : 0.f;
  }
  f32x16 acc[QT];
#pragma unroll
  for (int u = 0; u < QT; ++u)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[u][r] = 0.f;

  Stager<4, 1> sk;
  Stager<NCV, (32 * NCV + 255) / 256> sv;
  // one 32-key block; TAIL is compile-time so the per-element work has no branches
  auto block = [&](auto tail_c, const bf16_t* ks, const bf16_t* vs, int k0) {
    constexpr bool TAIL = decltype(tail_c)::value;
    f32x16 s[QT], dp[QT];
#pragma unroll
    for (int u = 0; u < QT; ++u)
#pragma unroll
      for (int r = 0; r < 16; ++r) { s[u][r] = 0.f; dp[u][r] = 0.f; }
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const bf16x8 ka = ld_row<4>(ks, lq, 16 * t + 8 * g);
#pragma unroll
      for (int u = 0; u < QT; ++u) s[u] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qb[u][t], s[u], 0, 0, 0);
    }
#pragma unroll
    for (int t = 0; t < DV / 16; ++t) {
      const bf16x8 va = ld_row<NCV>(vs, lq, 16 * t + 8 * g);
#pragma unroll
      for (int u = 0; u < QT; ++u) dp[u] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, db[u][t], dp[u], 0, 0, 0);
    }
#pragma unroll
    for (int u = 0; u < QT; ++u) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float p = exp2_(fmaf(s[u][r], kL2E, -lq2[u]));
        if (TAIL) p = k0 + acc_row(r, g) < L ? p : 0.f;
        s[u][r] = p * (dp[u][r] - dd[u]);
      }
    }
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const bf16x8 ka = ld_tr<4>(ks, t, 0, lane);
#pragma unroll
      for (int u = 0; u < QT; ++u)
        acc[u] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, pack_regs(s[u], t), acc[u], 0, 0, 0);
    }
  };
  auto run = [&]() {
    sk.load(K, DK, 0, Lp, tid);
    sv.load(V, DV, 0, Lp, tid);
    __syncthreads();
    sk.store(Ks[0], tid);
    sv.store(Vs[0], tid);
    __syncthreads();
    int buf = 0;
    for (int k0 = 0; k0 < Lp; k0 += 32) {
      const bool more = k0 + 32 < Lp;
      if (more) {
        sk.load(K, DK, k0 + 32, Lp, tid);
        sv.load(V, DV, k0 + 32, Lp, tid);
      }
      if (k0 + 32 > L)
        block(std::integral_constant<bool, true>(), Ks[buf], Vs[buf], k0);
      else
        block(std::integral_constant<bool, false>(), Ks[buf], Vs[buf], k0);
      if (more) {
        sk.store(Ks[buf ^ 1], tid);
        sv.store(Vs[buf ^ 1], tid);
      }
      __syncthreads();
      buf ^= 1;
    }
  };
  // invalid queries have zero Q and dO rows and lse2 0: their dS rows are
  // dropped at the store and their Dv is written as 0
#pragma unroll
  for (int u = 0; u < QT; ++u) {
    dd[u] = dd[u] + __shfl_xor(dd[u], 32, 64);
    const int q = qw + 32 * u + lq;
    if (g == 0 && q < HWp) Dv[(int64_t)b * HWp + q] = qv[u] ? dd[u] : 0.f;
  }
  run();
#pragma unroll
  for (int u = 0; u < QT; ++u) {
    const int q = qw + 32 * u + lq;
    if (!qv[u]) continue;
    bf16_t* row = dqkv + ((int64_t)b * HW + q) * Nqkv;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint2 v = make_uint2(f2bf2(acc[u][4 * i], acc[u][4 * i + 1]), f2bf2(acc[u][4 * i + 2], acc[u][4 * i + 3]));
      *reinterpret_cast<uint2*>(row + 8 * i + 4 * g) = v;
    }
  }
}

// ------------------------------------------------------------- dK, dV (key-owned)
// A wave owns one key tile (32 keys); a block of 4 waves 128 keys; the loop
// runs over 32-query blocks staged in LDS (Q, dO, lse2, Dv).
template <int DV>
__global__ __launch_bounds__(256, 2) void k_attn_dkv(const bf16_t* qkv, int Nqkv, const bf16_t* kp,
                                                     const bf16_t* vp, const bf16_t* dO, const float* lse2,
                                                     const float* Dv, int HW, int L, int Lp, int HWp, bf16_t* dk,
                                                     bf16_t* dvv) {
  constexpr int DK = 32, NT = DV / 32, NCV = DV / 8;
  __shared__ __attribute__((aligned(16))) bf16_t Qs[2][32 * DK];
  __shared__ __attribute__((aligned(16))) bf16_t Ds[2][32 * DV];
  __shared__ __attribute__((aligned(16))) float Ls[2][32], Dd[2][32];
  const int b = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 5, lk = lane & 31;
  const int key = blockIdx.x * 128 + (tid >> 6) * 32 + lk;
  const bf16_t* Q = qkv + (int64_t)b * HW * Nqkv;
  const bf16_t* DO = dO + (int64_t)b * HW * DV;
  const float* LS = lse2 + (int64_t)b * HWp;
  const float* DD = Dv + (int64_t)b * HWp;
  const bool kv = key < L;
  const int keyc = key < Lp ? key : Lp - 1;
  bf16x8 kb[2], vb[DV / 16];
#pragma unroll
  for (int t = 0; t < 2; ++t) kb[t] = ld8g(kp + ((int64_t)b * Lp + keyc) * DK + 16 * t + 8 * g);
#pragma unroll
  for (int t = 0; t < DV / 16; ++t) vb[t] = ld8g(vp + ((int64_t)b * Lp + keyc) * DV + 16 * t + 8 * g);
  f32x16 adk, adv[NT];
#pragma unroll
  for (int r = 0; r < 16; ++r) adk[r] = 0.f;
#pragma unroll
  for (int j = 0; j < NT; ++j)
#pragma unroll
    for (int r = 0; r < 16; ++r) adv[j][r] = 0.f;

  Stager<4, 1> sq;
  Stager<NCV, (32 * NCV + 255) / 256> sd;
  float sl = 0.f, sdd = 0.f;
  auto load = [&](int q0) {
    sq.load(Q, Nqkv, q0, HW, tid);
    sd.load(DO, DV, q0, HW, tid);
    if (tid < 32) {
      sl = LS[q0 + tid];
      sdd = DD[q0 + tid];
    }
  };
  auto store = [&](int bf) {
    sq.store(Qs[bf], tid);
    sd.store(Ds[bf], tid);
    if (tid < 32) {
      Ls[bf][tid] = sl;
      Dd[bf][tid] = sdd;
    }
  };
  load(0);
  store(0);
  __syncthreads();
  int buf = 0;
  for (int q0 = 0; q0 < HWp; q0 += 32) {
    const bool more = q0 + 32 < HWp;
    if (more) load(q0 + 32);
    const bf16_t* qs = Qs[buf];
    const bf16_t* ds = Ds[buf];
    f32x16 s, dp;
#pragma unroll
    for (int r = 0; r < 16; ++r) { s[r] = 0.f; dp[r] = 0.f; }
#pragma unroll
    for (int t = 0; t < 2; ++t) s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ld_row<4>(qs, lk, 16 * t + 8 * g), kb[t], s, 0, 0, 0);
#pragma unroll
    for (int t = 0; t < DV / 16; ++t)
      dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ld_row<NCV>(ds, lk, 16 * t + 8 * g), vb[t], dp, 0, 0, 0);
    f32x16 p;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float4 lv = *reinterpret_cast<const float4*>(&Ls[buf][8 * i + 4 * g]);
      const float4 dv4 = *reinterpret_cast<const float4*>(&Dd[buf][8 * i + 4 * g]);
      const float lsv[4] = {lv.x, lv.y, lv.z, lv.w}, dvv_[4] = {dv4.x, dv4.y, dv4.z, dv4.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = 4 * i + e;
        const float pr = kv ? exp2_(fmaf(s[r], kL2E, -lsv[e])) : 0.f;
        p[r] = pr;
        s[r] = pr * (dp[r] - dvv_[e]);
      }
    }
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const bf16x8 pb = pack_regs(p, t), sb = pack_regs(s, t);
#pragma unroll
      for (int j = 0; j < NT; ++j)
        adv[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ld_tr<NCV>(ds, t, 32 * j, lane), pb, adv[j], 0, 0, 0);
      adk = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ld_tr<4>(qs, t, 0, lane), sb, adk, 0, 0, 0);
    }
    if (more) store(buf ^ 1);
    __syncthreads();
    buf ^= 1;
  }
  if (key < Lp) {
    bf16_t* dkr = dk + ((int64_t)b * Lp + key) * DK;
    bf16_t* dvr = dvv + ((int64_t)b * Lp + key) * DV;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      *reinterpret_cast<uint2*>(dkr + 8 * i + 4 * g) =
          make_uint2(f2bf2(adk[4 * i], adk[4 * i + 1]), f2bf2(adk[4 * i + 2], adk[4 * i + 3]));
#pragma unroll
      for (int j = 0; j < NT; ++j)
        *reinterpret_cast<uint2*>(dvr + 32 * j + 8 * i + 4 * g) =
            make_uint2(f2bf2(adv[j][4 * i], adv[j][4 * i + 1]), f2bf2(adv[j][4 * i + 2], adv[j][4 * i + 3]));
    }
  }
}

// Max-pool backward: route dK / dV to the window's argmax (recomputed from
// the forward projections with the same tie rule), zeros elsewhere.
// its backward, 8 channels per thread: the gradient goes to the window's
// (first) maximum, zeros elsewhere
__global__ void k_attn_pool_bwd(const bf16_t* qkv, const bf16_t* dk, const bf16_t* dvv, int B, int H, int W,
                                int Nqkv, int dkw, int dvw, int Lp, bf16_t* dqkv) {
  const int ng = (dkw + dvw) / 8;
  const int L = (H / 2) * (W / 2);
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= B * L * ng) return;
  const int g = i % ng, t = i / ng;
  const int l = t % L, b = t / L;
  const int c = 8 * g;
  const int ph = l / (W / 2), pw = l - ph * (W / 2);
  int arg[8];
  float bv[8];
#pragma unroll
  for (int d = 0; d < 4; ++d) {
    const int h = 2 * ph + (d >> 1), w = 2 * pw + (d & 1);
    float v[8];
    unpack8(*reinterpret_cast<const uint4*>(qkv + ((int64_t)(b * H + h) * W + w) * Nqkv + dkw + c), v);
#pragma unroll
    for (int e = 0; e < 8; ++e)
      if (d == 0 || v[e] > bv[e]) {
        bv[e] = v[e];
        arg[e] = d;
      }
  }
  const uint4 gq = c < dkw ? *reinterpret_cast<const uint4*>(dk + ((int64_t)b * Lp + l) * dkw + c)
                           : *reinterpret_cast<const uint4*>(dvv + ((int64_t)b * Lp + l) * dvw + c - dkw);
  const uint32_t* gw = reinterpret_cast<const uint32_t*>(&gq);
#pragma unroll
  for (int d = 0; d < 4; ++d) {
    const int h = 2 * ph + (d >> 1), w = 2 * pw + (d & 1);
    uint32_t o[4];
#pragma unroll
    for (int k2 = 0; k2 < 4; ++k2) {
      const uint32_t lo = arg[2 * k2] == d ? (gw[k2] & 0xffffu) : 0u;
      const uint32_t hi = arg[2 * k2 + 1] == d ? (gw[k2] & 0xffff0000u) : 0u;
      o[k2] = lo | hi;
    }
    *reinterpret_cast<uint4*>(dqkv + ((int64_t)(b * H + h) * W + w) * Nqkv + dkw + c) = make_uint4(o[0], o[1], o[2], o[3]);
  }
}

// dgamma = <Wo (packed bf16, [Cp][dv]), dWo_raw (fp32, same layout)>
__global__ void k_attn_dgamma(const bf16_t* wo, const float* dwo, int64_t n, float* out) {
  __shared__ double sh[4];
  double s = 0.0;
  for (int64_t i = threadIdx.x; i < n; i += 256) s += (double)bf2f(wo[i]) * dwo[i];
  s = wave_sum_d(s);
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) *out = (float)(sh[0] + sh[1] + sh[2] + sh[3]);
}

// --------------------------------------------------------------- launchers
#define PG_DV_DISPATCH(dv, CALL)                                         \
  switch (dv) {                                                          \
    case 32: { constexpr int DVc = 32; CALL; break; }                    \
    case 64: { constexpr int DVc = 64; CALL; break; }                    \
    case 96: { constexpr int DVc = 96; CALL; break; }                    \
    case 128: { constexpr int DVc = 128; CALL; break; }                  \
    default: throw Error{-2, "attention: value width must be 32, 64, 96 or 128"}; \
  }

void attn_pool(hipStream_t st, const AttnDims& a, const void* qkv, void* kp, void* vp) {
  PG_CHECK(a.dk % 8 == 0 && a.dv % 8 == 0 && a.Nqkv % 8 == 0, "attention pool: 8-channel groups");
  const int64_t n = (int64_t)a.B * a.Lp * ((a.dk + a.dv) / 8);
  PG_CHECK(n < (1LL << 31) && (int64_t)a.B * a.H * a.W * a.Nqkv < (1LL << 31), "attention pool: size");
  hipLaunchKernelGGL(k_attn_pool, dim3((unsigned)cdiv(n, 256)), dim3(256), 0, st, (const bf16_t*)qkv, a.B, a.H,
                     a.W, a.Nqkv, a.dk, a.dv, a.Lp, (bf16_t*)kp, (bf16_t*)vp);
  PG_LAUNCH_CHECK();
}

static void check_dims(const AttnDims& a) {
  PG_CHECK(a.dk == 32 && a.Lp % 32 == 0 && a.HWp % 32 == 0 && a.Nqkv % 8 == 0, "attention: dims");
}

void attn_fwd_core(hipStream_t st, const AttnDims& a, const void* qkv, const void* kp, const void* vp, void* o,
                   float* o32, float* lse2) {
  check_dims(a);
  dim3 grid((unsigned)cdiv(a.HWp, 256), a.B);
  ProfScope prof(st);
  PG_DV_DISPATCH(a.dv, hipLaunchKernelGGL(k_attn_fwd<DVc>, grid, dim3(256), 0, st, (const bf16_t*)qkv, a.Nqkv,
                                          (const bf16_t*)kp, (const bf16_t*)vp, a.HW, a.L, a.Lp, a.HWp,
                                          (bf16_t*)o, o32, lse2));
  PG_LAUNCH_CHECK();
  prof.done("k_attn_fwd<" + std::to_string(a.dv) + ">", 2.0 * a.B * (double)a.HW * a.L * (a.dk + a.dv));
}

void attn_bwd_core(hipStream_t st, const AttnDims& a, const void* qkv, const void* dO, const float* o32,
                   const void* kp, const void* vp, const float* lse2, float* Dv, void* dk, void* dvv, void* dqkv) {
  check_dims(a);
  dim3 gk((unsigned)cdiv(a.Lp, 128), a.B);
  ProfScope prof(st);
  PG_DV_DISPATCH(a.dv, {
    dim3 gq((unsigned)cdiv(a.HWp, 128 * dq_tiles<DVc>()), a.B);
    hipLaunchKernelGGL(k_attn_dq<DVc>, gq, dim3(256), 0, st, (const bf16_t*)qkv, a.Nqkv, (const bf16_t*)kp,
                       (const bf16_t*)vp, (const bf16_t*)dO, o32, lse2, Dv, a.HW, a.L, a.Lp, a.HWp,
                       (bf16_t*)dqkv);
    hipLaunchKernelGGL(k_attn_dkv<DVc>, gk, dim3(256), 0, st, (const bf16_t*)qkv, a.Nqkv, (const bf16_t*)kp,
                       (const bf16_t*)vp, (const bf16_t*)dO, lse2, Dv, a.HW, a.L, a.Lp, a.HWp, (bf16_t*)dk,
                       (bf16_t*)dvv);
  });
  // executed: dQ pass S, dP, dQ; dK/dV pass S, dP, dV, dK
  prof.done("k_attn_bwd<" + std::to_string(a.dv) + ">",
            2.0 * a.B * (double)a.HW * a.L * (4 * a.dk + 3 * a.dv));
  const int64_t n = (int64_t)a.B * a.L * ((a.dk + a.dv) / 8);
  PG_CHECK(a.dv % 8 == 0 && n < (1LL << 31) && (int64_t)a.B * a.H * a.W * a.Nqkv < (1LL << 31),
           "attention pool: size");
  hipLaunchKernelGGL(k_attn_pool_bwd, dim3((unsigned)cdiv(n, 256)), dim3(256), 0, st, (const bf16_t*)qkv,
                     (const bf16_t*)dk, (const bf16_t*)dvv, a.B, a.H, a.W, a.Nqkv, a.dk, a.dv, a.Lp,
                     (bf16_t*)dqkv);
  PG_LAUNCH_CHECK();
}

void attn_dgamma(hipStream_t st, const void* wo, const float* dwo, int64_t n, float* out) {
  hipLaunchKernelGGL(k_attn_dgamma, dim3(1), dim3(256), 0, st, (const bf16_t*)wo, dwo, n, out);
  PG_LAUNCH_CHECK();
}

}  // namespace pg
