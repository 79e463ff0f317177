// Self-attention core on gfx950 (bf16 MFMA 32x32x16, fp32 softmax).
//
// Per image: queries theta (HW x dk), keys phi and values g max-pooled 2x2
// (L = HW/4 rows), scores S = Q K^T without scaling, softmax over keys,
// O = P V.  Flash-style: S is never stored.  Each wave owns 32 queries and
// computes the transposed score tile S^T = K Q^T, so that every lane holds
// one query's scores and the softmax max/sum reductions stay in-lane (plus
// one swap with the lane 32 apart).  The probabilities then feed the second
// product O^T = V^T P^T straight from registers: the B operand's 8 k-slots
// of lane group g are the keys {4g..4g+3, 8+4g..8+4g+3} (+16 per k-step),
// and V^T is read with the same key order.  The backward recomputes P from
// the saved log-sum-exp: one kernel owns queries (dQ), one owns keys (dK,
// dV), so no float atomics are needed.
//
// Layouts (bf16 unless noted), per image b, key count padded to Lp = 32k
// and query count to HWp = 32k with zeros:
//   qkv [HW][Nqkv]   projections, theta | phi | g at channel offsets 0, dk, 2dk
//   kp [Lp][dk], kt [dk][Lp], vp [Lp][dv], vt [dv][Lp]   pooled keys/values
//   qt [dk][HWp], dot [dv][HWp]                           transposed Q, dO
//   o, dO [HW][dv];  lse, Dv [HWp] fp32
#include "attn.hpp"

namespace pg {

typedef __bf16 bf16x4v __attribute__((ext_vector_type(4)));

PG_DEV bf16x8 ld8(const bf16_t* p) { return *reinterpret_cast<const bf16x8*>(p); }
PG_DEV bf16x8 ld4x2(const bf16_t* p0, const bf16_t* p1) {
  const uint2 a = *reinterpret_cast<const uint2*>(p0);
  const uint2 b = *reinterpret_cast<const uint2*>(p1);
  uint4 q = make_uint4(a.x, a.y, b.x, b.y);
  return *reinterpret_cast<bf16x8*>(&q);
}
PG_DEV bf16x8 pack_regs(const f32x16& v, int t) {
  float f[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) f[i] = v[8 * t + i];
  uint4 q = pack8(f);
  return *reinterpret_cast<bf16x8*>(&q);
}
PG_DEV bf16x8 zero8() {
  uint4 q = make_uint4(0, 0, 0, 0);
  return *reinterpret_cast<bf16x8*>(&q);
}
// row index (within a 32-tile) held by accumulator register r of lane group g
PG_DEV int acc_row(int r, int g) { return 8 * (r >> 2) + 4 * g + (r & 3); }

// ------------------------------------------------------------- pooling
// Max over each 2x2 window (first maximum in (dh, dw) row-major order wins)
// of the phi and g channels; writes K, K^T, V, V^T with zero padding.
__global__ void k_attn_pool(const bf16_t* qkv, int B, int H, int W, int Nqkv, int dk, int dv, int Lp,
                            bf16_t* kp, bf16_t* kt, bf16_t* vp, bf16_t* vt) {
  const int L = (H / 2) * (W / 2);
  const int nch = dk + dv;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (int64_t)B * Lp * nch) return;
  const int c = (int)(i % nch);
  const int64_t t = i / nch;
  const int l = (int)(t % Lp);
  const int b = (int)(t / Lp);
  bf16_t best = 0;
  if (l < L) {
    const int ph = l / (W / 2), pw = l % (W / 2);
    float bv = 0.f;
    for (int d = 0; d < 4; ++d) {
      const int h = 2 * ph + (d >> 1), w = 2 * pw + (d & 1);
      const bf16_t v = qkv[(((int64_t)b * H + h) * W + w) * Nqkv + dk + c];
      if (d == 0 || bf2f(v) > bv) { bv = bf2f(v); best = v; }
    }
  }
  if (c < dk) {
    kp[((int64_t)b * Lp + l) * dk + c] = best;
    kt[((int64_t)b * dk + c) * Lp + l] = best;
  } else {
    const int cv = c - dk;
    vp[((int64_t)b * Lp + l) * dv + cv] = best;
    vt[((int64_t)b * dv + cv) * Lp + l] = best;
  }
}

// dst[b][c][q] = src[b][q][c0 + c] for q < HW, 0 for HW <= q < HWp
__global__ void k_attn_transpose(const bf16_t* src, int ld, int c0, int C, int HW, int HWp, int B, bf16_t* dst) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (int64_t)B * C * HWp) return;
  const int q = (int)(i % HWp);
  const int64_t t = i / HWp;
  const int c = (int)(t % C);
  const int b = (int)(t / C);
  dst[i] = q < HW ? src[((int64_t)b * HW + q) * ld + c0 + c] : (bf16_t)0;
}

// ------------------------------------------------------------- forward
template <int DV>
__global__ __launch_bounds__(256) void k_attn_fwd(const bf16_t* qkv, int Nqkv, const bf16_t* kp,
                                                  const bf16_t* vt, int HW, int L, int Lp, int HWp,
                                                  bf16_t* o, float* lse) {
  constexpr int DK = 32, NT = DV / 32;
  const int b = blockIdx.y;
  const int lane = threadIdx.x & 63, g = lane >> 5, lq = lane & 31;
  const int q0 = (blockIdx.x * 4 + (threadIdx.x >> 6)) * 32;
  if (q0 >= HWp) return;
  const int q = q0 + lq;
  const bf16_t* Q = qkv + (int64_t)b * HW * Nqkv;
  const bf16_t* K = kp + (int64_t)b * Lp * DK;
  const bf16_t* VT = vt + (int64_t)b * DV * Lp;
  bf16x8 qb[2];
#pragma unroll
  for (int t = 0; t < 2; ++t) qb[t] = q < HW ? ld8(Q + (int64_t)q * Nqkv + 16 * t + 8 * g) : zero8();
  f32x16 acc[NT];
#pragma unroll
  for (int j = 0; j < NT; ++j)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[j][r] = 0.f;
  float m = -INFINITY, l = 0.f;
  for (int k0 = 0; k0 < Lp; k0 += 32) {
    f32x16 s;
#pragma unroll
    for (int r = 0; r < 16; ++r) s[r] = 0.f;
#pragma unroll
    for (int t = 0; t < 2; ++t)
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ld8(K + (int64_t)(k0 + lq) * DK + 16 * t + 8 * g), qb[t], s,
                                                  0, 0, 0);
    float mb = -INFINITY;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      if (k0 + acc_row(r, g) >= L) s[r] = -INFINITY;
      mb = fmaxf(mb, s[r]);
    }
    mb = fmaxf(mb, __shfl_xor(mb, 32, 64));
    const float mn = fmaxf(m, mb);
    const float alpha = __expf(m - mn);
    m = mn;
    float ls = 0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      s[r] = __expf(s[r] - mn);
      ls += s[r];
    }
    l = l * alpha + ls;
#pragma unroll
    for (int j = 0; j < NT; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[j][r] *= alpha;
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const bf16x8 pb = pack_regs(s, t);
#pragma unroll
      for (int j = 0; j < NT; ++j) {
        const bf16_t* vr = VT + (int64_t)(j * 32 + lq) * Lp + k0 + 16 * t + 4 * g;
        acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ld4x2(vr, vr + 8), pb, acc[j], 0, 0, 0);
      }
    }
  }
  const float lt = l + __shfl_xor(l, 32, 64);
  const float inv = 1.f / lt;
  if (q < HW) {
    bf16_t* orow = o + ((int64_t)b * HW + q) * DV;
#pragma unroll
    for (int j = 0; j < NT; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) orow[j * 32 + acc_row(r, g)] = f2bf(acc[j][r] * inv);
  }
  if (g == 0 && q < HWp) lse[(int64_t)b * HWp + q] = q < HW ? m + __logf(lt) : 0.f;
}

// D[q] = sum_c dO[q][c] O[q][c]
__global__ void k_attn_dvec(const bf16_t* dO, const bf16_t* O, int dv, int HW, int HWp, int B, float* D) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (int64_t)B * HWp) return;
  const int q = (int)(i % HWp);
  const int b = (int)(i / HWp);
  float s = 0.f;
  if (q < HW) {
    const int64_t base = ((int64_t)b * HW + q) * dv;
    for (int c = 0; c < dv; ++c) s = fmaf(bf2f(dO[base + c]), bf2f(O[base + c]), s);
  }
  D[i] = s;
}

// ------------------------------------------------------------- dQ (query-owned)
// S^T = K Q^T and dP^T = V dO^T for one 32-key block (lane = query)
template <int DV>
PG_DEV void score_tiles(const bf16_t* K, const bf16_t* V, const bf16x8* qb, const bf16x8* db, int k0, int lq,
                        int g, f32x16& s, f32x16& dp) {
#pragma unroll
  for (int r = 0; r < 16; ++r) { s[r] = 0.f; dp[r] = 0.f; }
#pragma unroll
  for (int t = 0; t < 2; ++t)
    s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ld8(K + (int64_t)(k0 + lq) * 32 + 16 * t + 8 * g), qb[t], s, 0, 0,
                                                0);
#pragma unroll
  for (int t = 0; t < DV / 16; ++t)
    dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ld8(V + (int64_t)(k0 + lq) * DV + 16 * t + 8 * g), db[t], dp, 0,
                                                 0, 0);
}

template <int DV>
__global__ __launch_bounds__(256) void k_attn_dq(const bf16_t* qkv, int Nqkv, const bf16_t* kp,
                                                 const bf16_t* kt, const bf16_t* vp, const bf16_t* dO,
                                                 const float* lse, float* Dv, int HW, int L, int Lp,
                                                 int HWp, bf16_t* dqkv) {
  constexpr int DK = 32;
  const int b = blockIdx.y;
  const int lane = threadIdx.x & 63, g = lane >> 5, lq = lane & 31;
  const int q0 = (blockIdx.x * 4 + (threadIdx.x >> 6)) * 32;
  if (q0 >= HWp) return;
  const int q = q0 + lq;
  const bool qv = q < HW;
  const bf16_t* Q = qkv + (int64_t)b * HW * Nqkv;
  const bf16_t* K = kp + (int64_t)b * Lp * DK;
  const bf16_t* KT = kt + (int64_t)b * DK * Lp;
  const bf16_t* V = vp + (int64_t)b * Lp * DV;
  const bf16_t* DO = dO + (int64_t)b * HW * DV;
  bf16x8 qb[2];
#pragma unroll
  for (int t = 0; t < 2; ++t) qb[t] = qv ? ld8(Q + (int64_t)q * Nqkv + 16 * t + 8 * g) : zero8();
  bf16x8 db[DV / 16];
#pragma unroll
  for (int t = 0; t < DV / 16; ++t) db[t] = qv ? ld8(DO + (int64_t)q * DV + 16 * t + 8 * g) : zero8();
  const float lq_ = qv ? lse[(int64_t)b * HWp + q] : 0.f;
  // pass 1: D[q] = sum_k P[q][k] dP[q][k]  (the softmax backward's row term,
  // by its definition, from the same P and dP that pass 2 uses)
  float dsum = 0.f;
  for (int k0 = 0; k0 < Lp; k0 += 32) {
    f32x16 s, dp;
    score_tiles<DV>(K, V, qb, db, k0, lq, g, s, dp);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const bool kv = k0 + acc_row(r, g) < L;
      dsum += (kv && qv) ? __expf(s[r] - lq_) * dp[r] : 0.f;
    }
  }
  const float dq_ = dsum + __shfl_xor(dsum, 32, 64);
  if (g == 0 && q < HWp) Dv[(int64_t)b * HWp + q] = qv ? dq_ : 0.f;
  // pass 2: dQ^T = K^T dS^T
  f32x16 acc;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[r] = 0.f;
  for (int k0 = 0; k0 < Lp; k0 += 32) {
    f32x16 s, dp;
    score_tiles<DV>(K, V, qb, db, k0, lq, g, s, dp);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const bool kv = k0 + acc_row(r, g) < L;
      const float p = (kv && qv) ? __expf(s[r] - lq_) : 0.f;
      s[r] = p * (dp[r] - dq_);
    }
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const bf16_t* kr = KT + (int64_t)lq * Lp + k0 + 16 * t + 4 * g;
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ld4x2(kr, kr + 8), pack_regs(s, t), acc, 0, 0, 0);
    }
  }
  if (qv) {
    bf16_t* row = dqkv + ((int64_t)b * HW + q) * Nqkv;
#pragma unroll
    for (int r = 0; r < 16; ++r) row[acc_row(r, g)] = f2bf(acc[r]);
  }
}

// ------------------------------------------------------------- dK, dV (key-owned)
template <int DV>
__global__ __launch_bounds__(256) void k_attn_dkv(const bf16_t* qkv, int Nqkv, const bf16_t* qt,
                                                  const bf16_t* kp, const bf16_t* vp, const bf16_t* dO,
                                                  const bf16_t* dOt, const float* lse, const float* Dv, int HW,
                                                  int L, int Lp, int HWp, bf16_t* dk, bf16_t* dvv) {
  constexpr int DK = 32, NT = DV / 32;
  const int b = blockIdx.y;
  const int lane = threadIdx.x & 63, g = lane >> 5, lk = lane & 31;
  const int k0 = (blockIdx.x * 4 + (threadIdx.x >> 6)) * 32;
  if (k0 >= Lp) return;
  const int key = k0 + lk;
  const bf16_t* Q = qkv + (int64_t)b * HW * Nqkv;
  const bf16_t* QT = qt + (int64_t)b * DK * HWp;
  const bf16_t* K = kp + (int64_t)b * Lp * DK;
  const bf16_t* V = vp + (int64_t)b * Lp * DV;
  const bf16_t* DO = dO + (int64_t)b * HW * DV;
  const bf16_t* DOT = dOt + (int64_t)b * DV * HWp;
  const float* LS = lse + (int64_t)b * HWp;
  const float* DD = Dv + (int64_t)b * HWp;
  bf16x8 kb[2], vb[DV / 16];
#pragma unroll
  for (int t = 0; t < 2; ++t) kb[t] = ld8(K + (int64_t)key * DK + 16 * t + 8 * g);
#pragma unroll
  for (int t = 0; t < DV / 16; ++t) vb[t] = ld8(V + (int64_t)key * DV + 16 * t + 8 * g);
  const bool kv = key < L;
  f32x16 adk, adv[NT];
#pragma unroll
  for (int r = 0; r < 16; ++r) adk[r] = 0.f;
#pragma unroll
  for (int j = 0; j < NT; ++j)
#pragma unroll
    for (int r = 0; r < 16; ++r) adv[j][r] = 0.f;
  for (int q0 = 0; q0 < HWp; q0 += 32) {
    const int qa = q0 + lk;     // the query this lane supplies to A operands
    const bool qav = qa < HW;
    f32x16 s, dp;
#pragma unroll
    for (int r = 0; r < 16; ++r) { s[r] = 0.f; dp[r] = 0.f; }
#pragma unroll
    for (int t = 0; t < 2; ++t)
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qav ? ld8(Q + (int64_t)qa * Nqkv + 16 * t + 8 * g) : zero8(),
                                                  kb[t], s, 0, 0, 0);
#pragma unroll
    for (int t = 0; t < DV / 16; ++t)
      dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qav ? ld8(DO + (int64_t)qa * DV + 16 * t + 8 * g) : zero8(),
                                                   vb[t], dp, 0, 0, 0);
    f32x16 p;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int qq = q0 + acc_row(r, g);
      const bool ok = kv && qq < HW;
      p[r] = ok ? __expf(s[r] - LS[qq]) : 0.f;
      s[r] = ok ? p[r] * (dp[r] - DD[qq]) : 0.f;
    }
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const bf16x8 pb = pack_regs(p, t), sb = pack_regs(s, t);
#pragma unroll
      for (int j = 0; j < NT; ++j) {
        const bf16_t* dr = DOT + (int64_t)(j * 32 + lk) * HWp + q0 + 16 * t + 4 * g;
        adv[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ld4x2(dr, dr + 8), pb, adv[j], 0, 0, 0);
      }
      const bf16_t* qr = QT + (int64_t)lk * HWp + q0 + 16 * t + 4 * g;
      adk = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ld4x2(qr, qr + 8), sb, adk, 0, 0, 0);
    }
  }
  bf16_t* dkr = dk + ((int64_t)b * Lp + key) * DK;
#pragma unroll
  for (int r = 0; r < 16; ++r) dkr[acc_row(r, g)] = f2bf(adk[r]);
  bf16_t* dvr = dvv + ((int64_t)b * Lp + key) * DV;
#pragma unroll
  for (int j = 0; j < NT; ++j)
#pragma unroll
    for (int r = 0; r < 16; ++r) dvr[j * 32 + acc_row(r, g)] = f2bf(adv[j][r]);
}

// Max-pool backward: route dK / dV to the window's argmax (recomputed from
// the forward projections with the same tie rule), zeros elsewhere.
__global__ void k_attn_pool_bwd(const bf16_t* qkv, const bf16_t* dk, const bf16_t* dvv, int B, int H, int W,
                                int Nqkv, int dkw, int dvw, int Lp, bf16_t* dqkv) {
  const int nch = dkw + dvw;
  const int L = (H / 2) * (W / 2);
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (int64_t)B * L * nch) return;
  const int c = (int)(i % nch);
  const int64_t t = i / nch;
  const int l = (int)(t % L);
  const int b = (int)(t / L);
  const int ph = l / (W / 2), pw = l % (W / 2);
  int arg = 0;
  float bv = 0.f;
  for (int d = 0; d < 4; ++d) {
    const int h = 2 * ph + (d >> 1), w = 2 * pw + (d & 1);
    const float v = bf2f(qkv[(((int64_t)b * H + h) * W + w) * Nqkv + dkw + c]);
    if (d == 0 || v > bv) { bv = v; arg = d; }
  }
  const bf16_t gv = c < dkw ? dk[((int64_t)b * Lp + l) * dkw + c] : dvv[((int64_t)b * Lp + l) * dvw + c - dkw];
  for (int d = 0; d < 4; ++d) {
    const int h = 2 * ph + (d >> 1), w = 2 * pw + (d & 1);
    dqkv[(((int64_t)b * H + h) * W + w) * Nqkv + dkw + c] = d == arg ? gv : (bf16_t)0;
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

void attn_pool(hipStream_t st, const AttnDims& a, const void* qkv, void* kp, void* kt, void* vp, void* vt) {
  const int64_t n = (int64_t)a.B * a.Lp * (a.dk + a.dv);
  hipLaunchKernelGGL(k_attn_pool, dim3((unsigned)cdiv(n, 256)), dim3(256), 0, st, (const bf16_t*)qkv, a.B, a.H,
                     a.W, a.Nqkv, a.dk, a.dv, a.Lp, (bf16_t*)kp, (bf16_t*)kt, (bf16_t*)vp, (bf16_t*)vt);
  PG_LAUNCH_CHECK();
}

void attn_transpose(hipStream_t st, const AttnDims& a, const void* src, int ld, int c0, int C, void* dst) {
  const int64_t n = (int64_t)a.B * C * a.HWp;
  hipLaunchKernelGGL(k_attn_transpose, dim3((unsigned)cdiv(n, 256)), dim3(256), 0, st, (const bf16_t*)src, ld, c0,
                     C, a.HW, a.HWp, a.B, (bf16_t*)dst);
  PG_LAUNCH_CHECK();
}

void attn_fwd_core(hipStream_t st, const AttnDims& a, const void* qkv, const void* kp, const void* vt, void* o,
                   float* lse) {
  dim3 grid((unsigned)cdiv(a.HWp, 128), a.B);
  ProfScope prof(st);
  PG_DV_DISPATCH(a.dv, hipLaunchKernelGGL(k_attn_fwd<DVc>, grid, dim3(256), 0, st, (const bf16_t*)qkv, a.Nqkv,
                                          (const bf16_t*)kp, (const bf16_t*)vt, a.HW, a.L, a.Lp, a.HWp,
                                          (bf16_t*)o, lse));
  PG_LAUNCH_CHECK();
  prof.done("k_attn_fwd<" + std::to_string(a.dv) + ">", 2.0 * a.B * (double)a.HW * a.L * (a.dk + a.dv));
}

void attn_bwd_core(hipStream_t st, const AttnDims& a, const void* qkv, const void* o, const void* dO,
                   const void* kp, const void* kt, const void* vp, const void* qt, const void* dOt,
                   const float* lse, float* Dv, void* dk, void* dvv, void* dqkv) {
  dim3 gq((unsigned)cdiv(a.HWp, 128), a.B), gk((unsigned)cdiv(a.Lp, 128), a.B);
  ProfScope prof(st);
  PG_DV_DISPATCH(a.dv, {
    hipLaunchKernelGGL(k_attn_dq<DVc>, gq, dim3(256), 0, st, (const bf16_t*)qkv, a.Nqkv, (const bf16_t*)kp,
                       (const bf16_t*)kt, (const bf16_t*)vp, (const bf16_t*)dO, lse, Dv, a.HW, a.L, a.Lp, a.HWp,
                       (bf16_t*)dqkv);
    hipLaunchKernelGGL(k_attn_dkv<DVc>, gk, dim3(256), 0, st, (const bf16_t*)qkv, a.Nqkv, (const bf16_t*)qt,
                       (const bf16_t*)kp, (const bf16_t*)vp, (const bf16_t*)dO, (const bf16_t*)dOt, lse, Dv, a.HW,
                       a.L, a.Lp, a.HWp, (bf16_t*)dk, (bf16_t*)dvv);
  });
  // dQ: 2 passes of S and dP plus dQ; dK/dV: S, dP, dV, dK
  prof.done("k_attn_bwd<" + std::to_string(a.dv) + ">",
            2.0 * a.B * (double)a.HW * a.L * (3 * a.dk + 4 * a.dv));
  const int64_t n = (int64_t)a.B * a.L * (a.dk + a.dv);
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
