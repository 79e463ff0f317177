// Self-attention block executor: fused theta|phi|g projection (one 1x1
// implicit-GEMM conv), max-pool, flash attention core, output projection
// with the gamma-scaled residual in its epilogue; and the backward.
#include "attn.hpp"
#include "blocks.hpp"

namespace pg {

static AttnDims dims(const Attn& t) {
  AttnDims a;
  a.B = t.B; a.H = t.H; a.W = t.W; a.HW = t.H * t.W; a.L = (t.H / 2) * (t.W / 2);
  a.Lp = (int)cdiv(a.L, 32) * 32; a.HWp = (int)cdiv(a.HW, 32) * 32;
  a.dk = t.dk; a.dv = t.dv; a.Nqkv = t.Nqkv;
  return a;
}

void Attn::plan_saved(Arena& a) {
  Cp = (int)cpad(C);
  dk = 32;
  dv = (int)cpad(C / 2);
  Nqkv = 2 * dk + dv;
  const AttnDims d = dims(*this);
  const int64_t rows[4] = {C / 8, C / 8, C / 2, C};
  const int64_t cols[4] = {C, C, C, C / 2};
  for (int i = 0; i < 4; ++i) {
    sn[i].u = a.f32(rows[i]);
    sn[i].v = a.f32(cols[i]);
    sn[i].sigma = a.f32(1);
  }
  wqkv = a.bytes((size_t)Nqkv * Cp * 2);
  wo = a.bytes((size_t)Cp * dv * 2);
  qkv = a.bytes((size_t)B * d.HW * Nqkv * 2);
  kp = a.bytes((size_t)B * d.Lp * dk * 2);
  vp = a.bytes((size_t)B * d.Lp * dv * 2);
  o = a.bytes((size_t)B * d.HW * dv * 2);
  o32 = a.f32((size_t)B * d.HWp * dv);
  lse = a.f32((size_t)B * d.HWp);
}

struct AWsB {
  void *wdq, *wdo, *dO, *dk, *dvv, *dqkv, *wg;
  float *Dv, *dwq, *dwo, *part;
  size_t wg_bytes;
};

static AWsB a_carve_b(const Attn& t, Arena& a, int n_cu) {
  const AttnDims d = dims(t);
  AWsB w;
  const int64_t M = (int64_t)t.B * d.HW;
  w.wdq = a.bytes((size_t)t.Cp * t.Nqkv * 2);
  w.wdo = a.bytes((size_t)t.dv * t.Cp * 2);
  w.dO = a.bytes((size_t)M * t.dv * 2);
  w.dk = a.bytes((size_t)t.B * d.Lp * t.dk * 2);
  w.dvv = a.bytes((size_t)t.B * d.Lp * t.dv * 2);
  w.dqkv = a.bytes((size_t)M * t.Nqkv * 2);
  w.Dv = a.f32((size_t)t.B * d.HWp);
  w.dwq = a.f32((size_t)t.Nqkv * t.Cp);
  w.dwo = a.f32((size_t)t.Cp * t.dv);
  w.part = a.f32((size_t)kSnbParts * kSnGroupMax);
  w.wg_bytes = std::max(conv_wgrad_ws(false, M, 1, t.dv, t.Cp, n_cu), conv_wgrad_ws(false, M, 1, t.Cp, t.Nqkv, n_cu));
  w.wg = a.bytes(w.wg_bytes);
  return w;
}

size_t Attn::ws_size(int n_cu) const {
  const int64_t rc[4][2] = {{C / 8, C}, {C / 8, C}, {C / 2, C}, {C, C / 2}};
  const size_t sn_b = sn_group_ws(rc, 4);
  Arena b(nullptr);
  a_carve_b(*this, b, n_cu);
  return std::max(align256(sn_b), b.off);
}

static const char* kASN[4] = {"theta", "phi", "g", "o"};

void Attn::sn_jobs(const Params& P, std::vector<SnJob>& out) {
  for (int i = 0; i < 4; ++i) out.push_back(sn_job(P, kASN[i], sn[i]));
}

void Attn::pack_jobs(const Params& P, std::vector<PackJob>& out) {
  out.push_back({P.w("theta"), sn[0].sigma, wqkv, C / 8, C, 1, dk, Cp, kPackFwd});
  out.push_back({P.w("phi"), sn[1].sigma, (char*)wqkv + (size_t)dk * Cp * 2, C / 8, C, 1, dk, Cp, kPackFwd});
  out.push_back({P.w("g"), sn[2].sigma, (char*)wqkv + (size_t)2 * dk * Cp * 2, C / 2, C, 1, dv, Cp, kPackFwd});
  out.push_back({P.w("o"), sn[3].sigma, wo, C, C / 2, 1, Cp, dv, kPackFwd});
}

void Attn::prep(hipStream_t st, const Params& P, void* sn_ws) {
  std::vector<SnJob> sj;
  sn_jobs(P, sj);
  sn_power_iter_all(st, sj.data(), (int)sj.size(), npi, sn_eps, sn_ws);
  std::vector<PackJob> pk;
  pack_jobs(P, pk);
  pack_all(st, false, pk.data(), (int)pk.size());
}

void Attn::fwd(const Exec& ex, const Params& P, const void* x, void* y, bool for_bwd) {
  const AttnDims d = dims(*this);
  if (!prepped) prep(ex.st, P, ex.ws);
  ConvIn in;
  in.x = x; in.B = B; in.Hx = H; in.Wx = W; in.C = Cp;
  ConvOut po;
  po.y = qkv; po.yC = Nqkv; po.n_real = Nqkv;
  conv_fwd(ex.st, false, in, H, W, 1, wqkv, Nqkv, po);
  attn_pool(ex.st, d, qkv, kp, vp);
  attn_fwd_core(ex.st, d, qkv, kp, vp, o, for_bwd ? o32 : nullptr, lse);
  ConvIn oi;
  oi.x = o; oi.B = B; oi.Hx = H; oi.Wx = W; oi.C = dv;
  ConvOut oo;
  oo.y = y; oo.yC = Cp; oo.n_real = C; oo.acc_scale = P.w("gamma");
  oo.res = x; oo.res_mode = R_SAME; oo.resC = Cp;
  conv_fwd(ex.st, false, oi, H, W, 1, wo, Cp, oo);
}

void Attn::bwd(const Exec& ex, const Params& P, const void* x, const void* dy, void* dx, bool wgrad) {
  const AttnDims d = dims(*this);
  Arena a(ex.ws);
  AWsB w = a_carve_b(*this, a, ex.n_cu);
  const int64_t M = (int64_t)B * d.HW;
  const float* gamma = P.w("gamma");
  // output projection: raw dWo = sum dy (x) O; dgamma = <Wo, raw dWo>
  GradIn gdy;
  gdy.g = dy; gdy.Hs = H; gdy.Ws = W; gdy.C = Cp;
  ConvIn ao;
  ao.x = o; ao.B = B; ao.Hx = H; ao.Wx = W; ao.C = dv;
  if (wgrad) {
    conv_wgrad(ex.st, false, gdy, ao, H, W, 1, Cp, w.dwo, w.wg, w.wg_bytes, ex.n_cu);
    attn_dgamma(ex.st, wo, w.dwo, (int64_t)Cp * dv, P.gr("gamma"));
  }
  // dO = gamma * dy Wo
  pack_weight(ex.st, false, P.w("o"), sn[3].sigma, C, C / 2, 1, Cp, dv, true, w.wdo);
  ConvIn di;
  di.x = dy; di.B = B; di.Hx = H; di.Wx = W; di.C = Cp;
  ConvOut dOo;
  dOo.y = w.dO; dOo.yC = dv; dOo.n_real = dv; dOo.acc_scale = gamma;
  conv_fwd(ex.st, false, di, H, W, 1, w.wdo, dv, dOo);
  attn_bwd_core(ex.st, d, qkv, w.dO, o32, kp, vp, lse, w.Dv, w.dk, w.dvv, w.dqkv);
  // projections
  GradIn gq;
  gq.g = w.dqkv; gq.Hs = H; gq.Ws = W; gq.C = Nqkv;
  ConvIn ax;
  ax.x = x; ax.B = B; ax.Hx = H; ax.Wx = W; ax.C = Cp;
  if (wgrad) conv_wgrad(ex.st, false, gq, ax, H, W, 1, Nqkv, w.dwq, w.wg, w.wg_bytes, ex.n_cu);
  pack_weight_t(ex.st, false, P.w("theta"), sn[0].sigma, C / 8, C, Cp, dk, Nqkv, 0, w.wdq);
  pack_weight_t(ex.st, false, P.w("phi"), sn[1].sigma, C / 8, C, Cp, dk, Nqkv, dk, w.wdq);
  pack_weight_t(ex.st, false, P.w("g"), sn[2].sigma, C / 2, C, Cp, dv, Nqkv, 2 * dk, w.wdq);
  ConvIn qi;
  qi.x = w.dqkv; qi.B = B; qi.Hx = H; qi.Wx = W; qi.C = Nqkv;
  ConvOut xo;
  xo.y = dx; xo.yC = Cp; xo.n_real = C; xo.res = dy; xo.res_mode = R_SAME; xo.resC = Cp;
  conv_fwd(ex.st, false, qi, H, W, 1, w.wdq, Cp, xo);
  (void)M;
  if (!wgrad) return;
  const SnBwdJob jobs[4] = {sn_bwd_job(P, "theta", sn[0], w.dwq, 1, Cp, nullptr),
                            sn_bwd_job(P, "phi", sn[1], w.dwq + (size_t)dk * Cp, 1, Cp, nullptr),
                            sn_bwd_job(P, "g", sn[2], w.dwq + (size_t)2 * dk * Cp, 1, Cp, nullptr),
                            sn_bwd_job(P, "o", sn[3], w.dwo, 1, dv, gamma)};
  sn_bwd_group(ex.st, jobs, 4, w.part);
}

}  // namespace pg
