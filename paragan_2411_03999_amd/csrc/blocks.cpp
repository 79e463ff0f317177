// Residual-block executors: the order of kernel launches for the BigGAN
// generator and discriminator blocks, forward and backward.
#include "blocks.hpp"
#include "heads.hpp"

namespace pg {

const Entry& Layout::get(const std::string& name) const {
  for (const auto& x : e)
    if (x.name == name) return x;
  throw Error{-1, "layout: no parameter named " + name};
}

void Layout::add_prefixed(const std::string& prefix, const Layout& sub) {
  for (const auto& x : sub.e) add(prefix + x.name, x.shape, x.sn);
}

Layout gblock_layout(int cin, int cout, int dc) {
  Layout L;
  L.add("bn1.gain", {cin, dc}, true);
  L.add("bn1.bias", {cin, dc}, true);
  L.add("conv1.w", {cout, 3, 3, cin}, true);
  L.add("conv1.b", {cout}, false);
  L.add("bn2.gain", {cout, dc}, true);
  L.add("bn2.bias", {cout, dc}, true);
  L.add("conv2.w", {cout, 3, 3, cout}, true);
  L.add("conv2.b", {cout}, false);
  L.add("sc.w", {cout, 1, 1, cin}, true);
  L.add("sc.b", {cout}, false);
  return L;
}

Layout dblock_layout(int cin, int cout, bool lsc) {
  Layout L;
  L.add("conv1.w", {cout, 3, 3, cin}, true);
  L.add("conv1.b", {cout}, false);
  L.add("conv2.w", {cout, 3, 3, cout}, true);
  L.add("conv2.b", {cout}, false);
  if (lsc) {
    L.add("sc.w", {cout, 1, 1, cin}, true);
    L.add("sc.b", {cout}, false);
  }
  return L;
}

Layout attn_layout(int c) {
  Layout L;
  L.add("theta", {c / 8, 1, 1, c}, true);
  L.add("phi", {c / 8, 1, 1, c}, true);
  L.add("g", {c / 2, 1, 1, c}, true);
  L.add("o", {c, 1, 1, c / 2}, true);
  L.add("gamma", {1}, false);
  return L;
}

static int64_t cols_of(const Entry& e) { return e.numel() / e.shape[0]; }

void sn_forward(const Exec& ex, const Params& P, const std::string& name, SNSlot& s, int npi, float eps) {
  const SnJob j = sn_job(P, name, s);
  sn_power_iter_group(ex.st, &j, 1, npi, eps, ex.ws);
}

SnJob sn_job(const Params& P, const std::string& name, SNSlot& s) {
  const Entry& e = P.ent(name);
  return SnJob{P.p + e.offset, e.shape[0], cols_of(e), P.u + e.u_offset, s.v, s.sigma, s.u};
}

size_t sn_ws_all(const Layout& L) {
  size_t t = 0;
  for (const Entry& e : L.e)
    if (e.sn) t += sn_ws_bytes(e.shape[0], cols_of(e));
  return t;
}

size_t sn_group_ws(const int64_t (*rc)[2], int n) {
  size_t t = 0;
  for (int i = 0; i < n; ++i) t += sn_ws_bytes(rc[i][0], rc[i][1]);
  return t;
}

SnBwdJob sn_bwd_job(const Params& P, const std::string& name, const SNSlot& s, const float* dwp, int R, int Cp,
                    const float* scale) {
  const Entry& e = P.ent(name);
  return SnBwdJob{dwp, P.p + e.offset, s.u, s.v, s.sigma, scale, P.g + e.offset, (int)e.shape[0],
                  (int)(cols_of(e) / (R * R)), R, Cp};
}

static void plan_sn(Arena& a, SNSlot& s, int64_t rows, int64_t cols) {
  s.u = a.f32(rows);
  s.v = a.f32(cols);
  s.sigma = a.f32(1);
}

static size_t esz(bool f32) { return f32 ? 4 : 2; }

// ======================================================================
// generator block
// ======================================================================
static const char* kGSN[7] = {"bn1.gain", "bn1.bias", "conv1.w", "bn2.gain", "bn2.bias", "conv2.w", "sc.w"};

void GBlock::plan_saved(Arena& a) {
  Cip = (int)cpad(cin);
  Cop = (int)cpad(cout);
  const int64_t cols[7] = {dc, dc, 9LL * cin, dc, dc, 9LL * cout, cin};
  const int64_t rows[7] = {cin, cin, cout, cout, cout, cout, cout};
  for (int i = 0; i < 7; ++i) plan_sn(a, sn[i], rows[i], cols[i]);
  const size_t e = esz(f32);
  // bf16: conv1 over the upsample as four 2x2 sub-pixel filters (16 taps)
  wp1 = a.bytes((size_t)Cop * (f32 ? 9 : 16) * Cip * e);
  wp2 = a.bytes((size_t)Cop * 9 * Cop * e);
  wpsc = a.bytes((size_t)Cop * Cip * e);
  if (keep_dgrad) {
    wd1s = a.bytes((size_t)Cip * (f32 ? 9 : 16) * Cop * e);
    wd2s = a.bytes((size_t)Cop * 9 * Cop * e);
    wdscs = a.bytes((size_t)Cip * Cop * e * (f32 ? 1 : 4));
  }
  mean1 = a.f32(Cip); rstd1 = a.f32(Cip);
  gain1 = a.f32((size_t)B * Cip); bias1 = a.f32((size_t)B * Cip); scale1 = a.f32((size_t)B * Cip);
  mean2 = a.f32(Cop); rstd2 = a.f32(Cop);
  gain2 = a.f32((size_t)B * Cop); bias2 = a.f32((size_t)B * Cop); scale2 = a.f32((size_t)B * Cop);
  h1 = a.bytes((size_t)B * 4 * H * W * Cop * e);
  a1 = a.bytes((size_t)B * H * W * Cip * e);
  a2 = a.bytes((size_t)B * 4 * H * W * Cop * e);
}

struct GWsF {
  void* sn;
  void* bn;
  float* skip;
};
struct GWsB {
  void *wd1, *wd2, *wdsc;
  float *dwp1, *dwp2, *dwpsc, *dlin[4];
  void* wg;
  size_t wg_bytes;
  void* cs;
  float *dxs, *da2, *da1;
  void* dh1;
  float *dg1, *db1, *dg2, *db2, *part, *lin;
  void* bnb;
};

static size_t g_sn_ws(const GBlock& g) {
  const int64_t rc[7][2] = {{g.cin, g.dc}, {g.cin, g.dc}, {g.cout, 9LL * g.cin}, {g.cout, g.dc},
                            {g.cout, g.dc}, {g.cout, 9LL * g.cout}, {g.cout, g.cin}};
  return sn_group_ws(rc, 7);
}

static GWsF g_carve_f(const GBlock& g, Arena& a) {
  GWsF w;
  const int64_t M1 = (int64_t)g.B * g.H * g.W, M2 = 4 * M1;
  w.sn = a.bytes(g_sn_ws(g));
  w.bn = a.bytes(std::max(bn_stats_ws_bytes(M1, g.cin), bn_stats_ws_bytes(M2, g.cout)));
  w.skip = a.f32((size_t)M1 * g.Cop);
  return w;
}

static GWsB g_carve_b(const GBlock& g, Arena& a, int n_cu) {
  GWsB w;
  const int64_t M1 = (int64_t)g.B * g.H * g.W, M2 = 4 * M1;
  const size_t e = esz(g.f32);
  // bf16: conv1's data gradient as the stride-2 4x4 filter (16 taps)
  w.wd1 = a.bytes((size_t)g.Cip * (g.f32 ? 9 : 16) * g.Cop * e);
  w.wd2 = a.bytes((size_t)g.Cop * 9 * g.Cop * e);
  w.wdsc = a.bytes((size_t)g.Cip * g.Cop * e * (g.f32 ? 1 : 4));
  w.dwp1 = a.f32((size_t)g.Cop * 9 * g.Cip);
  w.dwp2 = a.f32((size_t)g.Cop * 9 * g.Cop);
  w.dwpsc = a.f32((size_t)g.Cop * g.Cip);
  for (int i = 0; i < 4; ++i) w.dlin[i] = a.f32((size_t)(i < 2 ? g.cin : g.cout) * g.dc);
  w.wg_bytes = std::max({conv_wgrad_ws(g.f32, M2, 3, g.Cip, g.Cop, n_cu),
                         conv_wgrad_ws(g.f32, M2, 3, g.Cop, g.Cop, n_cu),
                         conv_wgrad_ws(g.f32, M2, 1, g.Cip, g.Cop, n_cu),
                         g.f32 ? (size_t)0 : wgrad_sub_ws(M1, g.Cip, g.Cop, n_cu)});
  w.wg = a.bytes(w.wg_bytes);
  w.cs = a.bytes(colsum_ws_bytes(M2, g.Cop));
  w.dxs = a.f32((size_t)M1 * g.Cip);
  w.da2 = a.f32((size_t)M2 * g.Cop);
  w.da1 = a.f32((size_t)M2 * g.Cip);
  w.dh1 = a.bytes((size_t)M2 * g.Cop * e);
  w.dg1 = a.f32((size_t)g.B * g.Cip); w.db1 = a.f32((size_t)g.B * g.Cip);
  w.dg2 = a.f32((size_t)g.B * g.Cop); w.db2 = a.f32((size_t)g.B * g.Cop);
  w.part = a.f32((size_t)kSnbParts * kSnGroupMax);
  w.lin = (float*)a.bytes(cbn_linear_bwd_ws_bytes(g.B, g.dc));
  w.bnb = a.bytes(std::max(bn_bwd_ws_bytes(g.B, 4 * g.H * g.W, g.cout), bn_bwd_ws_bytes(g.B, g.H * g.W, g.cin)));
  return w;
}

size_t GBlock::ws_size(int n_cu) const {
  Arena a(nullptr), b(nullptr);
  g_carve_f(*this, a);
  g_carve_b(*this, b, n_cu);
  return std::max(a.off, b.off);
}

// the data-gradient weight packs of a G block into (wd1, wd2, wdsc)
static void g_pack_dgrad_jobs(const GBlock& g, const Params& P, void* wd1, void* wd2, void* wdsc,
                              std::vector<PackJob>& out) {
  // unnormalised: the data-gradient convs divide by sigma
  out.push_back({P.w("conv1.w"), nullptr, wd1, g.cout, g.cin, 3, g.Cop, g.Cip, g.f32 ? kPackDgrad : kPackDgradSum4});
  out.push_back({P.w("conv2.w"), nullptr, wd2, g.cout, g.cout, 3, g.Cop, g.Cop, kPackDgrad});
  out.push_back({P.w("sc.w"), nullptr, wdsc, g.cout, g.cin, 1, g.Cop, g.Cip, g.f32 ? kPackDgrad : kPackDgradRep4});
}
static void g_pack_dgrad(const GBlock& g, hipStream_t st, const Params& P, void* wd1, void* wd2, void* wdsc) {
  std::vector<PackJob> pk;
  g_pack_dgrad_jobs(g, P, wd1, wd2, wdsc, pk);
  pack_all(st, g.f32, pk.data(), (int)pk.size());
}

void GBlock::sn_jobs(const Params& P, std::vector<SnJob>& out) {
  for (int i = 0; i < 7; ++i) out.push_back(sn_job(P, kGSN[i], sn[i]));
}

void GBlock::pack_jobs(const Params& P, bool for_bwd, std::vector<PackJob>& out) {
  // the filters are packed unnormalised (the stored bf16 values do not
  // depend on sigma); each conv divides its accumulator by its sigma
  out.push_back({P.w("conv1.w"), nullptr, wp1, cout, cin, 3, Cop, Cip, f32 ? kPackFwd : kPackSub});
  out.push_back({P.w("conv2.w"), nullptr, wp2, cout, cout, 3, Cop, Cop, kPackFwd});
  out.push_back({P.w("sc.w"), nullptr, wpsc, cout, cin, 1, Cop, Cip, kPackFwd});
  if (for_bwd && keep_dgrad) {
    g_pack_dgrad_jobs(*this, P, wd1s, wd2s, wdscs, out);
    dgrad_ready = true;
  }
}

void GBlock::prep(hipStream_t st, const Params& P, void* sn_ws, bool for_bwd) {
  std::vector<SnJob> sj;
  sn_jobs(P, sj);
  sn_power_iter_all(st, sj.data(), (int)sj.size(), npi, sn_eps, sn_ws);
  std::vector<PackJob> pk;
  pack_jobs(P, for_bwd, pk);
  pack_all(st, f32, pk.data(), (int)pk.size());
}

void GBlock::fwd(const Exec& ex, const Params& P, const void* x, const float* cond, void* y) {
  Arena a(ex.ws);
  GWsF w = g_carve_f(*this, a);
  if (!prepped) prep(ex.st, P, w.sn);
  const int64_t M1 = (int64_t)B * H * W, M2 = 4 * M1;
  // cBN1 statistics and tables
  bn_stats(ex.st, f32, x, M1, cin, Cip, bn_eps, mean1, rstd1, w.bn);
  cbn_tables(ex.st, cond, dc, P.w("bn1.gain"), P.w("bn1.bias"), sn[0].sigma, sn[1].sigma, nullptr, nullptr,
             rstd1, B, cin, Cip, gain1, bias1, scale1);
  // h1 = conv3x3(up2(a1)) + b1, a1 = relu(cbn1(x)) (stored once, bf16)
  bn_apply(ex.st, f32, x, M1, H * W, cin, Cip, mean1, scale1, bias1, Cip, true, a1);
  ConvIn in;
  in.x = a1; in.B = B; in.Hx = H; in.Wx = W; in.C = Cip; in.gather = G_UP2;
  ConvOut o;
  o.y = h1; o.y_f32 = f32; o.yC = Cop; o.n_real = cout; o.bias = P.w("conv1.b"); o.acc_div = sn[2].sigma;
  if (!f32) {
    // bf16: the four sub-pixel 2x2 convs over a1 itself
    in.gather = G_SUB;
    conv_fwd(ex.st, f32, in, H, W, 2, wp1, Cop, o);
  } else {
    conv_fwd(ex.st, f32, in, 2 * H, 2 * W, 3, wp1, Cop, o);
  }
  // cBN2
  bn_stats(ex.st, f32, h1, M2, cout, Cop, bn_eps, mean2, rstd2, w.bn);
  cbn_tables(ex.st, cond, dc, P.w("bn2.gain"), P.w("bn2.bias"), sn[3].sigma, sn[4].sigma, nullptr, nullptr,
             rstd2, B, cout, Cop, gain2, bias2, scale2);
  // skip at low resolution (conv1x1 commutes with the nearest upsample)
  ConvIn si;
  si.x = x; si.B = B; si.Hx = H; si.Wx = W; si.C = Cip;
  ConvOut so;
  so.y = w.skip; so.y_f32 = 1; so.yC = Cop; so.n_real = cout; so.bias = P.w("sc.b"); so.acc_div = sn[6].sigma;
  conv_fwd(ex.st, f32, si, H, W, 1, wpsc, Cop, so);
  // y = conv3x3(a2) + b2 + up2(skip), a2 = relu(cbn2(h1))
  bn_apply(ex.st, f32, h1, M2, 4 * H * W, cout, Cop, mean2, scale2, bias2, Cop, true, a2);
  ConvIn i2;
  i2.x = a2; i2.B = B; i2.Hx = 2 * H; i2.Wx = 2 * W; i2.C = Cop;
  ConvOut o2;
  o2.y = y; o2.y_f32 = f32; o2.yC = Cop; o2.n_real = cout; o2.bias = P.w("conv2.b"); o2.acc_div = sn[5].sigma;
  o2.res = w.skip; o2.res_f32 = 1; o2.res_mode = R_HALF; o2.resC = Cop;
  conv_fwd(ex.st, f32, i2, 2 * H, 2 * W, 3, wp2, Cop, o2);
}

// The weight gradients of a block backward (and their bias column sums)
// read only the output gradients and the saved activations: with ex.side
// they run on that stream, forked from ex.st once their gradient is ready,
// while the data gradients continue on ex.st; the join comes before the SN
// backward, which reads them.  The kernels are the same either way, so are
// the results.
struct WgSide {
  const Exec& ex;
  hipStream_t sw;
  explicit WgSide(const Exec& e) : ex(e), sw(e.side ? e.side : e.st) {}
  void fork() const {
    if (!ex.side) return;
    PG_HIP(hipEventRecord(ex.ev_fork, ex.st));
    PG_HIP(hipStreamWaitEvent(sw, ex.ev_fork, 0));
  }
  void join() const {
    if (!ex.side) return;
    PG_HIP(hipEventRecord(ex.ev_join, sw));
    PG_HIP(hipStreamWaitEvent(ex.st, ex.ev_join, 0));
  }
};

void GBlock::bwd(const Exec& ex, const Params& P, const void* x, const float* cond, const void* dy, void* dx,
                 float* dcond, bool dcond_acc) {
  Arena a(ex.ws);
  GWsB w = g_carve_b(*this, a, ex.n_cu);
  const int64_t M1 = (int64_t)B * H * W, M2 = 4 * M1;
  const int H2 = 2 * H, W2 = 2 * W;
  // the data-gradient weights: packed by prep, or here
  void *wd1 = w.wd1, *wd2 = w.wd2, *wdsc = w.wdsc;
  if (dgrad_ready) {
    wd1 = wd1s; wd2 = wd2s; wdsc = wdscs;
    dgrad_ready = false;
  } else {
    g_pack_dgrad(*this, ex.st, P, wd1, wd2, wdsc);
  }
  const WgSide side(ex);
  const hipStream_t sw = side.sw;
  side.fork();
  // conv2: dW2, db2
  GradIn gdy;
  gdy.g = dy; gdy.Hs = H2; gdy.Ws = W2; gdy.C = Cop;
  ConvIn ia2;
  ia2.x = a2; ia2.B = B; ia2.Hx = H2; ia2.Wx = W2; ia2.C = Cop;
  conv_wgrad(sw, f32, gdy, ia2, H2, W2, 3, Cop, w.dwp2, w.wg, w.wg_bytes, ex.n_cu);
  colsum(sw, f32, dy, M2, cout, Cop, 1.f, P.gr("conv2.b"), w.cs);
  // skip: dWsc at full resolution against up2(x); dbsc = db2
  ConvIn ax;
  ax.x = x; ax.B = B; ax.Hx = H; ax.Wx = W; ax.C = Cip; ax.gather = G_UP2;
  conv_wgrad(sw, f32, gdy, ax, H2, W2, 1, Cop, w.dwpsc, w.wg, w.wg_bytes, ex.n_cu);
  // both biases add to the block output: their gradients are the same column sum of dy
  PG_HIP(hipMemcpyAsync(P.gr("sc.b"), P.gr("conv2.b"), (size_t)cout * 4, hipMemcpyDeviceToDevice, sw));
  // dx_skip = Wsc^T sum2x2(dy)   (low resolution, fp32); in bf16 one
  // stride-2 2x2 conv with Wsc^T on every tap
  ConvIn dsp;
  dsp.x = dy; dsp.B = B; dsp.Hx = H2; dsp.Wx = W2; dsp.C = Cop; dsp.gather = f32 ? G_POOL2 : G_S2;
  ConvOut dso;
  dso.y = w.dxs; dso.y_f32 = 1; dso.yC = Cip; dso.n_real = cin; dso.acc_div = sn[6].sigma;
  conv_fwd(ex.st, f32, dsp, H, W, f32 ? 1 : 2, wdsc, Cip, dso);
  // da2 = conv2^T dy (fp32)
  ConvIn d2;
  d2.x = dy; d2.B = B; d2.Hx = H2; d2.Wx = W2; d2.C = Cop;
  ConvOut d2o;
  d2o.y = w.da2; d2o.y_f32 = 1; d2o.yC = Cop; d2o.n_real = cout; d2o.acc_div = sn[5].sigma;
  conv_fwd(ex.st, f32, d2, H2, W2, 3, wd2, Cop, d2o);
  // cBN2 backward (through the ReLU) -> dh1
  bn_bwd(ex.st, f32, w.da2, false, h1, B, H2, W2, cout, Cop, mean2, rstd2, gain2, bias2, Cop, nullptr, w.dh1,
         w.dg2, w.db2, Cop, w.bnb);
  side.fork();
  // conv1: dW1, db1
  GradIn gdh;
  gdh.g = w.dh1; gdh.Hs = H2; gdh.Ws = W2; gdh.C = Cop;
  ConvIn ia1;
  ia1.x = a1; ia1.B = B; ia1.Hx = H; ia1.Wx = W; ia1.C = Cip; ia1.gather = G_UP2;
  if (!f32) {
    // bf16: the four sub-pixel 2x2 forms over a1 itself, folded onto the 3x3 filter
    ConvIn src = ia1;
    src.gather = G_DIRECT;
    wgrad_sub(sw, gdh, src, Cop, w.dwp1, w.wg, w.wg_bytes, ex.n_cu);
  } else {
    conv_wgrad(sw, f32, gdh, ia1, H2, W2, 3, Cop, w.dwp1, w.wg, w.wg_bytes, ex.n_cu);
  }
  colsum(sw, f32, w.dh1, M2, cout, Cop, 1.f, P.gr("conv1.b"), w.cs);
  // da1 = the 2x2 sum (the upsample's adjoint) of conv1^T dh1: in bf16 one
  // stride-2 4x4 conv straight to the low resolution; in fp32 at 2x
  // resolution, summed by the BN backward
  ConvIn d1;
  d1.x = w.dh1; d1.B = B; d1.Hx = H2; d1.Wx = W2; d1.C = Cop;
  ConvOut d1o;
  d1o.y = w.da1; d1o.y_f32 = 1; d1o.yC = Cip; d1o.n_real = cin; d1o.acc_div = sn[2].sigma;
  if (!f32) {
    d1.gather = G_S2;
    conv_fwd(ex.st, f32, d1, H, W, 4, wd1, Cip, d1o);
  } else {
    conv_fwd(ex.st, f32, d1, H2, W2, 3, wd1, Cip, d1o);
  }
  bn_bwd(ex.st, f32, w.da1, f32, x, B, H, W, cin, Cip, mean1, rstd1, gain1, bias1, Cip, w.dxs, dx, w.dg1,
         w.db1, Cip, w.bnb);
  // conditional-BN linear maps (+ their SN) and dcond
  struct Lin { const char* name; float* dgb; int C; int slot; };
  const Lin lins[4] = {{"bn1.gain", w.dg1, cin, 0}, {"bn1.bias", w.db1, cin, 1},
                       {"bn2.gain", w.dg2, cout, 3}, {"bn2.bias", w.db2, cout, 4}};
  const int Cps[4] = {Cip, Cip, Cop, Cop};
  SnBwdJob jobs[7];
  for (int i = 0; i < 4; ++i) {
    const Lin& l = lins[i];
    cbn_linear_bwd(ex.st, l.dgb, B, l.C, Cps[i], cond, dc, P.w(l.name), sn[l.slot].sigma, w.dlin[i], dcond,
                   dcond_acc || i > 0, w.lin);
    jobs[i] = sn_bwd_job(P, l.name, sn[l.slot], w.dlin[i], 1, dc, nullptr);
  }
  jobs[4] = sn_bwd_job(P, "conv1.w", sn[2], w.dwp1, 3, Cip, nullptr);
  jobs[5] = sn_bwd_job(P, "conv2.w", sn[5], w.dwp2, 3, Cop, nullptr);
  jobs[6] = sn_bwd_job(P, "sc.w", sn[6], w.dwpsc, 1, Cip, nullptr);
  side.join();
  sn_bwd_group(ex.st, jobs, 7, w.part);
}

// ======================================================================
// discriminator block
// ======================================================================
void DBlock::plan_saved(Arena& a) {
  PG_CHECK(!im2col || (9 * cin <= 32 && !f32 && !preact), "dblock: 3x3-patch input needs 9 cin <= 32, bf16, no ReLU");
  Cip = (int)cpad(im2col ? 9 * cin : cin);
  Cop = (int)cpad(cout);
  Ho = down ? H / 2 : H;
  Wo = down ? W / 2 : W;
  plan_sn(a, sn[0], cout, 9LL * cin);
  plan_sn(a, sn[1], cout, 9LL * cout);
  if (lsc) plan_sn(a, sn[2], cout, cin);
  const size_t e = esz(f32);
  wp1 = a.bytes((size_t)Cop * 9 * Cip * e);
  // a downsampling bf16 block keeps conv2 as the pre-pooled stride-2 4x4 filter
  wp2 = a.bytes((size_t)Cop * (s2conv() ? 16 : 9) * Cop * e);
  if (keep_dgrad) {
    wd1s = a.bytes((size_t)Cip * 9 * Cop * e);
    wd2s = a.bytes((size_t)Cop * (subdgrad() ? 16 : 9) * Cop * e);
    wdscs = lsc ? a.bytes((size_t)Cip * Cop * e) : nullptr;
  }
  if (lsc) wpsc = a.bytes((size_t)Cop * Cip * e);
  h = a.bytes((size_t)B * H * W * Cop * e);
  // the pooled block input, operand of the downsampling 1x1 skip
  xp = lsc && down ? a.bytes((size_t)B * Ho * Wo * Cip * e) : nullptr;
}

struct DWsF {
  void* sn;
  float* skip;
};
struct DWsB {
  void *wd1, *wd2, *wdsc;
  float *dwp1, *dwp2, *dwpsc, *dwp2s;
  void* wg;
  size_t wg_bytes;
  void* cs;
  void* dh;
  float* dxs;
  float* part;
  float* dcol;   // im2col: gradient of the 3x3 patches
};

static DWsF d_carve_f(const DBlock& d, Arena& a) {
  DWsF w;
  const int64_t rc[3][2] = {{d.cout, 9LL * d.cin}, {d.cout, 9LL * d.cout}, {d.cout, d.cin}};
  w.sn = a.bytes(sn_group_ws(rc, d.lsc ? 3 : 2));
  w.skip = d.lsc ? a.f32((size_t)d.B * d.Ho * d.Wo * d.Cop) : nullptr;
  return w;
}

static DWsB d_carve_b(const DBlock& d, Arena& a, int n_cu) {
  DWsB w;
  const int64_t M = (int64_t)d.B * d.H * d.W, Mo = (int64_t)d.B * d.Ho * d.Wo;
  const size_t e = esz(d.f32);
  w.wd1 = a.bytes((size_t)d.Cip * 9 * d.Cop * e);
  // with the pooled conv2: its data gradient as four sub-pixel 2x2 filters
  w.wd2 = a.bytes((size_t)d.Cop * (d.subdgrad() ? 16 : 9) * d.Cop * e);
  w.wdsc = d.lsc ? a.bytes((size_t)d.Cip * d.Cop * e) : nullptr;
  w.dwp1 = a.f32((size_t)d.Cop * 9 * d.Cip);
  w.dwp2 = a.f32((size_t)d.Cop * 9 * d.Cop);
  w.dwpsc = d.lsc ? a.f32((size_t)d.Cop * d.Cip) : nullptr;
  // the pooled conv2's gradient in its stride-2 4x4 form, folded to 3x3 after
  w.dwp2s = d.s2conv() ? a.f32((size_t)d.Cop * 16 * d.Cop) : nullptr;
  w.wg_bytes = std::max(conv_wgrad_ws(d.f32, M, 3, d.Cip, d.Cop, n_cu), conv_wgrad_ws(d.f32, M, 3, d.Cop, d.Cop, n_cu));
  if (d.s2conv()) w.wg_bytes = std::max(w.wg_bytes, conv_wgrad_ws(d.f32, Mo, 4, d.Cop, d.Cop, n_cu));
  if (d.lsc) w.wg_bytes = std::max(w.wg_bytes, conv_wgrad_ws(d.f32, Mo, 1, d.Cip, d.Cop, n_cu));
  w.wg = a.bytes(w.wg_bytes);
  w.cs = a.bytes(colsum_ws_bytes(M, d.Cop));
  w.dh = a.bytes((size_t)M * d.Cop * e);
  w.dxs = d.lsc ? a.f32((size_t)Mo * d.Cip) : nullptr;
  w.part = a.f32((size_t)kSnbParts * kSnGroupMax);
  w.dcol = d.im2col ? a.f32((size_t)M * d.Cip) : nullptr;
  return w;
}

size_t DBlock::ws_size(int n_cu) const {
  Arena a(nullptr), b(nullptr);
  d_carve_f(*this, a);
  d_carve_b(*this, b, n_cu);
  return std::max(a.off, b.off);
}

// the data-gradient weight packs of a D block into (wd1, wd2, wdsc)
static void d_pack_dgrad_jobs(const DBlock& d, const Params& P, void* wd1, void* wd2, void* wdsc,
                              std::vector<PackJob>& out) {
  const int R1 = d.im2col ? 1 : 3, K1 = d.im2col ? 9 * d.cin : d.cin, ksc = d.im2col ? 4 * d.cin : 0;
  // unnormalised: the data-gradient convs divide by sigma
  out.push_back({P.w("conv1.w"), nullptr, wd1, d.cout, K1, R1, d.Cop, d.Cip, kPackDgrad});
  out.push_back({P.w("conv2.w"), nullptr, wd2, d.cout, d.cout, 3, d.Cop, d.Cop,
                 d.subdgrad() ? kPackSubDgrad : kPackDgrad});
  if (d.lsc) out.push_back({P.w("sc.w"), nullptr, wdsc, d.cout, d.cin, 1, d.Cop, d.Cip, kPackDgrad, ksc});
}
static void d_pack_dgrad(const DBlock& d, hipStream_t st, const Params& P, void* wd1, void* wd2, void* wdsc) {
  std::vector<PackJob> pk;
  d_pack_dgrad_jobs(d, P, wd1, wd2, wdsc, pk);
  pack_all(st, d.f32, pk.data(), (int)pk.size());
}

void DBlock::sn_jobs(const Params& P, std::vector<SnJob>& out) {
  out.push_back(sn_job(P, "conv1.w", sn[0]));
  out.push_back(sn_job(P, "conv2.w", sn[1]));
  if (lsc) out.push_back(sn_job(P, "sc.w", sn[2]));
}

void DBlock::pack_jobs(const Params& P, bool for_bwd, std::vector<PackJob>& out) {
  // with 3x3-patch input, conv1 is a 1x1 filter over the 9 cin patch
  // channels (the [Cout][3][3][cin] weight read as [Cout][9 cin]) and the
  // skip's 1x1 filter sits on the centre tap's channels 4 cin ..
  const int R1 = im2col ? 1 : 3, K1 = im2col ? 9 * cin : cin, ksc = im2col ? 4 * cin : 0;
  // packed unnormalised; each conv divides its accumulator by its sigma
  out.push_back({P.w("conv1.w"), nullptr, wp1, cout, K1, R1, Cop, Cip, kPackFwd});
  out.push_back({P.w("conv2.w"), nullptr, wp2, cout, cout, 3, Cop, Cop, s2conv() ? kPackPool4 : kPackFwd});
  if (lsc) out.push_back({P.w("sc.w"), nullptr, wpsc, cout, cin, 1, Cop, Cip, kPackFwd, ksc});
  if (for_bwd && keep_dgrad) {
    d_pack_dgrad_jobs(*this, P, wd1s, wd2s, wdscs, out);
    dgrad_ready = true;
  }
}

void DBlock::prep(hipStream_t st, const Params& P, void* sn_ws, bool for_bwd) {
  std::vector<SnJob> sj;
  sn_jobs(P, sj);
  sn_power_iter_all(st, sj.data(), (int)sj.size(), npi, sn_eps, sn_ws);
  std::vector<PackJob> pk;
  pack_jobs(P, for_bwd, pk);
  pack_all(st, f32, pk.data(), (int)pk.size());
}

void DBlock::fwd(const Exec& ex, const Params& P, const void* x, void* y) {
  Arena a(ex.ws);
  DWsF w = d_carve_f(*this, a);
  if (!prepped) prep(ex.st, P, w.sn);
  const int R1 = im2col ? 1 : 3, K1 = im2col ? 9 * cin : cin, ksc = im2col ? 4 * cin : 0;
  // h = conv3x3([relu](x)) + b1
  ConvIn i1;
  i1.x = x; i1.B = B; i1.Hx = H; i1.Wx = W; i1.C = Cip; i1.relu = preact; i1.c_real = K1;
  ConvOut o1;
  o1.y = h; o1.y_f32 = f32; o1.yC = Cop; o1.n_real = cout; o1.bias = P.w("conv1.b"); o1.acc_div = sn[0].sigma;
  conv_fwd(ex.st, f32, i1, H, W, R1, wp1, Cop, o1);
  // skip = conv1x1([avgpool](x)) + bsc, fp32
  if (lsc) {
    ConvIn si;
    si.x = x; si.B = B; si.Hx = H; si.Wx = W; si.C = Cip; si.c_real = cin;
    if (down) {
      avgpool2(ex.st, f32, x, B, H, W, Cip, xp);
      si.x = xp; si.Hx = Ho; si.Wx = Wo;
    }
    ConvOut so;
    so.y = w.skip; so.y_f32 = 1; so.yC = Cop; so.n_real = cout; so.bias = P.w("sc.b"); so.acc_div = sn[2].sigma;
    conv_fwd(ex.st, f32, si, Ho, Wo, 1, wpsc, Cop, so);
  }
  // y = [avgpool](conv3x3(relu(h)) + b2) + skip; with downsampling in bf16 the
  // pool is folded into the filter: a stride-2 4x4 conv at the pooled pixels
  ConvIn i2;
  i2.x = h; i2.B = B; i2.Hx = H; i2.Wx = W; i2.C = Cop; i2.relu = 1;
  ConvOut o2;
  o2.y = y; o2.y_f32 = f32; o2.yC = Cop; o2.n_real = cout; o2.bias = P.w("conv2.b"); o2.pool = down;
  o2.acc_div = sn[1].sigma;
  o2.res_mode = R_SAME; o2.resC = Cop;
  if (lsc) { o2.res = w.skip; o2.res_f32 = 1; }
  else { o2.res = x; o2.res_f32 = f32; }
  if (s2conv()) {
    i2.gather = G_S2;
    o2.pool = 0;
    conv_fwd(ex.st, f32, i2, Ho, Wo, 4, wp2, Cop, o2);
  } else {
    conv_fwd(ex.st, f32, i2, H, W, 3, wp2, Cop, o2);
  }
}

void DBlock::bwd(const Exec& ex, const Params& P, const void* x, const void* dy, void* dx, bool dx_f32,
                 bool wgrad) {
  Arena a(ex.ws);
  DWsB w = d_carve_b(*this, a, ex.n_cu);
  const int64_t M = (int64_t)B * H * W, Mo = (int64_t)B * Ho * Wo;
  const int R1 = im2col ? 1 : 3, K1 = im2col ? 9 * cin : cin, ksc = im2col ? 4 * cin : 0;
  // the data-gradient weights: packed by prep, or here
  void *wd1 = w.wd1, *wd2 = w.wd2, *wdsc = w.wdsc;
  if (dgrad_ready) {
    wd1 = wd1s; wd2 = wd2s; wdsc = wdscs;
    dgrad_ready = false;
  } else {
    d_pack_dgrad(*this, ex.st, P, wd1, wd2, wdsc);
  }
  const WgSide side(ex);
  const hipStream_t sw = side.sw;
  if (wgrad) side.fork();
  // conv2 (its output gradient is dy, or dy/4 spread over 2x2 when pooled)
  GradIn g2;
  g2.g = dy; g2.Hs = Ho; g2.Ws = Wo; g2.C = Cop;
  if (down) { g2.gather = G_UP2; g2.gscale = 0.25f; }
  ConvIn a2;
  a2.x = h; a2.B = B; a2.Hx = H; a2.Wx = W; a2.C = Cop; a2.relu = 1;
  if (wgrad) {
    if (s2conv()) {
      // the gradient of the stride-2 4x4 form: pooled dy against relu(h) read
      // at stride 2, then folded back onto the 3x3 filter
      GradIn g2s;
      g2s.g = dy; g2s.Hs = Ho; g2s.Ws = Wo; g2s.C = Cop;
      ConvIn a2s = a2;
      a2s.gather = G_S2;
      conv_wgrad(sw, f32, g2s, a2s, Ho, Wo, 4, Cop, w.dwp2s, w.wg, w.wg_bytes, ex.n_cu);
      fold_pool4_wgrad(sw, w.dwp2s, Cop, Cop, w.dwp2);
    } else {
      conv_wgrad(sw, f32, g2, a2, H, W, 3, Cop, w.dwp2, w.wg, w.wg_bytes, ex.n_cu);
    }
    colsum(sw, f32, dy, Mo, cout, Cop, 1.f, P.gr("conv2.b"), w.cs);
  }
  // dh = (conv2^T dc2) * [h > 0]
  ConvIn d2;
  d2.x = dy; d2.B = B; d2.Hx = Ho; d2.Wx = Wo; d2.C = Cop;
  if (down) { d2.gather = G_UP2; d2.gscale = 0.25f; }
  ConvOut d2o;
  d2o.y = w.dh; d2o.y_f32 = f32; d2o.yC = Cop; d2o.n_real = cout; d2o.acc_div = sn[1].sigma;
  d2o.mask = h; d2o.mask_f32 = f32; d2o.maskC = Cop;
  if (subdgrad()) {
    // conv2^T over up2(dy) / 4 as the four sub-pixel 2x2 convs over dy
    d2.gather = G_SUB;
    conv_fwd(ex.st, f32, d2, Ho, Wo, 2, wd2, Cop, d2o);
  } else {
    conv_fwd(ex.st, f32, d2, H, W, 3, wd2, Cop, d2o);
  }
  // conv1
  GradIn g1;
  g1.g = w.dh; g1.Hs = H; g1.Ws = W; g1.C = Cop;
  ConvIn a1;
  a1.x = x; a1.B = B; a1.Hx = H; a1.Wx = W; a1.C = Cip; a1.relu = preact; a1.c_real = K1;
  if (wgrad) {
    side.fork();   // dh is ready
    conv_wgrad(sw, f32, g1, a1, H, W, R1, Cop, w.dwp1, w.wg, w.wg_bytes, ex.n_cu);
    colsum(sw, f32, w.dh, M, cout, Cop, 1.f, P.gr("conv1.b"), w.cs);
  }
  // skip
  if (lsc) {
    GradIn gs;
    gs.g = dy; gs.Hs = Ho; gs.Ws = Wo; gs.C = Cop;
    ConvIn as;
    as.x = x; as.B = B; as.Hx = H; as.Wx = W; as.C = Cip; as.c_real = cin;
    if (down) { as.x = xp; as.Hx = Ho; as.Wx = Wo; }
    if (wgrad) {
      conv_wgrad(sw, f32, gs, as, Ho, Wo, 1, Cop, w.dwpsc, w.wg, w.wg_bytes, ex.n_cu);
      // both biases add to the block output (after the pool): the same column sum of dy
      PG_HIP(hipMemcpyAsync(P.gr("sc.b"), P.gr("conv2.b"), (size_t)cout * 4, hipMemcpyDeviceToDevice, sw));
    }
    if (dx) {
      ConvIn ds;
      ds.x = dy; ds.B = B; ds.Hx = Ho; ds.Wx = Wo; ds.C = Cop;
      ConvOut dso;
      dso.y = w.dxs; dso.y_f32 = 1; dso.yC = Cip; dso.n_real = ksc + cin; dso.acc_div = sn[2].sigma;
      conv_fwd(ex.st, f32, ds, Ho, Wo, 1, wdsc, Cip, dso);
    }
  }
  if (dx) {
    ConvIn d1;
    d1.x = w.dh; d1.B = B; d1.Hx = H; d1.Wx = W; d1.C = Cop;
    ConvOut d1o;
    // with 3x3-patch input: the patch gradient (fp32), folded onto the image after
    d1o.y = im2col ? (void*)w.dcol : dx; d1o.y_f32 = dx_f32 || f32 || im2col; d1o.yC = Cip;
    d1o.acc_div = sn[0].sigma;
    d1o.n_real = im2col ? K1 : cin;
    if (preact) { d1o.mask = x; d1o.mask_f32 = f32; d1o.maskC = Cip; }
    if (lsc) {
      d1o.res = w.dxs; d1o.res_f32 = 1; d1o.resC = Cip;
      d1o.res_mode = down ? R_HALF : R_SAME;
      d1o.res_scale = down ? 0.25f : 1.f;
    } else {
      d1o.res = dy; d1o.res_f32 = f32; d1o.resC = Cop; d1o.res_mode = R_SAME;
    }
    conv_fwd(ex.st, f32, d1, H, W, R1, wd1, Cip, d1o);
    if (im2col) im2col_grad(ex.st, w.dcol, B, H, W, (float*)dx);
  }
  if (!wgrad) return;
  side.join();
  const SnBwdJob jobs[3] = {sn_bwd_job(P, "conv1.w", sn[0], w.dwp1, R1, Cip, nullptr),
                            sn_bwd_job(P, "conv2.w", sn[1], w.dwp2, 3, Cop, nullptr),
                            lsc ? sn_bwd_job(P, "sc.w", sn[2], w.dwpsc + ksc, 1, Cip, nullptr) : SnBwdJob{}};
  sn_bwd_group(ex.st, jobs, lsc ? 3 : 2, w.part);
}

}  // namespace pg
