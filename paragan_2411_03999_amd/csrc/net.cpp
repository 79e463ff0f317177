// BigGAN generator / discriminator executors and the G+D train step.
//
// One training iteration (Numerical Optimizations, "Asynchronous Update
// Scheme": the D:G ratio is adjustable; here n_D discriminator updates per
// generator update) runs entirely on the context's stream:
//   D step k:  G forward on (z_k, y_k) writing the fake half of the D batch,
//              D forward / hinge / backward on concat(real_k, fake_k) --
//              inputs that share a weight go through one batched pass
//              (Implementation, "Hardware-Aware Layout Transformation") --
//              then Adam on D;
//   G step:    G forward, D forward, hinge, D backward for the input
//              gradient only, G backward, Adam on G.
// Only one host synchronisation per call: the losses at the end.
#include "net.hpp"

#include <cstdio>

namespace pg {

Arch arch_from(const paragan_biggan_desc* d) {
  Arch a;
  a.img = d->img; a.ch = d->ch; a.n_g = d->n_g; a.n_d = d->n_d; a.attn_res = d->attn_res;
  a.n_classes = d->n_classes; a.dz = d->dz; a.sd = d->shared_dim;
  a.zc = d->n_g >= 0 ? d->dz / (d->n_g + 1) : 0;
  a.dc = a.sd + a.zc;
  for (int i = 0; i <= d->n_g && i < 10; ++i) a.g_mult.push_back(d->g_mult[i]);
  for (int j = 0; j < d->n_d && j < 10; ++j) {
    a.d_mult.push_back(d->d_mult[j]);
    a.d_down.push_back(d->d_down[j]);
  }
  a.npi = d->n_power_iter; a.bn_eps = d->bn_eps; a.sn_eps = d->sn_eps;
  return a;
}

std::vector<DSpec> d_specs(const Arch& a) {
  std::vector<DSpec> v;
  int res = a.img, cin = 3;
  bool placed = false;
  for (int j = 0; j < a.n_d; ++j) {
    DSpec s;
    s.cin = cin; s.cout = a.d_mult[j] * a.ch; s.H = res; s.W = res;
    s.preact = j > 0; s.down = a.d_down[j] != 0; s.lsc = s.cin != s.cout || s.down;
    res = s.down ? res / 2 : res;
    s.attn = !placed && a.attn_res > 0 && res == a.attn_res;
    placed = placed || s.attn;
    v.push_back(s);
    cin = s.cout;
  }
  return v;
}

static bool attn_width_ok(int C) {
  const int dv = (int)cpad(C / 2);
  return C % 8 == 0 && C / 8 <= 32 && (dv == 32 || dv == 64 || dv == 96 || dv == 128);
}

void check_arch(const paragan_biggan_desc* d) {
  if (!d) throw Error{-1, "biggan: desc is NULL"};
  PG_CHECK(d->n_g >= 1 && d->n_g <= 9, "biggan: n_g must be in [1, 9]");
  PG_CHECK(d->n_d >= 1 && d->n_d <= 10, "biggan: n_d must be in [1, 10]");
  PG_CHECK(d->ch >= 1 && d->B >= 1 && d->n_classes >= 1 && d->shared_dim >= 1, "biggan: ch, B, n_classes, shared_dim >= 1");
  PG_CHECK(d->img == (4 << d->n_g), "biggan: img must equal 4 * 2^n_g");
  PG_CHECK(d->dz >= d->n_g + 1 && d->dz % (d->n_g + 1) == 0, "biggan: dz must split into n_g + 1 equal chunks");
  for (int i = 0; i <= d->n_g; ++i) PG_CHECK(d->g_mult[i] >= 1, "biggan: g_mult entries must be >= 1");
  for (int j = 0; j < d->n_d; ++j) PG_CHECK(d->d_mult[j] >= 1, "biggan: d_mult entries must be >= 1");
  PG_CHECK(d->n_power_iter >= 1 && d->bn_eps > 0 && d->sn_eps > 0, "biggan: bad eps / n_power_iter");
  for (const paragan_optim* o : {&d->opt_g, &d->opt_d})
    PG_CHECK((o->kind == PARAGAN_ADAM || o->kind == PARAGAN_ADABELIEF) && o->lr >= 0 && o->beta1 >= 0 &&
                 o->beta1 < 1 && o->beta2 >= 0 && o->beta2 < 1 && o->eps > 0,
             "biggan: bad optimiser settings (kind Adam or AdaBelief, lr >= 0, 0 <= beta < 1, eps > 0)");
  PG_CHECK((int64_t)2 * d->B * d->img * d->img < (1LL << 31), "biggan: batch too large");
  const Arch a = arch_from(d);
  int res = a.img;
  for (const DSpec& s : d_specs(a)) {
    PG_CHECK(!s.down || (res % 2 == 0 && res >= 2), "biggan: a pooling D block needs an even resolution");
    res = s.down ? res / 2 : res;
    if (s.attn) PG_CHECK(attn_width_ok(s.cout) && res % 2 == 0, "biggan: unsupported D attention width");
  }
  for (int i = 0; i < a.n_g; ++i)
    if ((4 << (i + 1)) == a.attn_res)
      PG_CHECK(attn_width_ok(a.g_mult[i + 1] * a.ch), "biggan: unsupported G attention width");
  PG_CHECK(ghead_shape_ok(a.img, a.g_mult[a.n_g] * a.ch),
           "biggan: the generator output layer takes at most 128 (padded) input channels");
}

Layout g_layout(const Arch& a) {
  Layout L;
  const int c0 = a.g_mult[0] * a.ch;
  L.add("shared", {a.n_classes, a.sd}, false);
  L.add("linear.w", {16LL * c0, a.zc}, true);
  L.add("linear.b", {16LL * c0}, false);
  for (int i = 0; i < a.n_g; ++i) {
    const int cout = a.g_mult[i + 1] * a.ch;
    L.add_prefixed("g" + std::to_string(i) + ".", gblock_layout(a.g_mult[i] * a.ch, cout, a.dc));
    if ((4 << (i + 1)) == a.attn_res) L.add_prefixed("attn.", attn_layout(cout));
  }
  L.add_prefixed("", gout_layout(a.g_mult[a.n_g] * a.ch));
  return L;
}

Layout d_layout(const Arch& a) {
  Layout L;
  const auto specs = d_specs(a);
  for (int j = 0; j < (int)specs.size(); ++j) {
    const DSpec& s = specs[j];
    L.add_prefixed("d" + std::to_string(j) + ".", dblock_layout(s.cin, s.cout, s.lsc));
    if (s.attn) L.add_prefixed("attn.", attn_layout(s.cout));
  }
  const int c = a.d_mult[a.n_d - 1] * a.ch;
  L.add("head.w", {1, c}, true);
  L.add("head.b", {1}, false);
  L.add("embed", {a.n_classes, c}, true);
  return L;
}

static Params sub(const Params& P, const std::string& prefix) {
  Params q = P;
  q.prefix = prefix;
  return q;
}

static void plan_slot(Arena& s, SNSlot& slot, int64_t rows, int64_t cols) {
  slot.u = s.f32(rows);
  slot.v = s.f32(cols);
  slot.sigma = s.f32(1);
}

// =================================================================== G
void GNet::plan_saved(Arena& s) {
  const Arch& a = a_;
  const int c0 = a.g_mult[0] * a.ch;
  plan_slot(s, lin_, 16LL * c0, a.zc);
  cond_.clear();
  for (int i = 0; i < a.n_g; ++i) cond_.push_back(s.f32((size_t)B_ * a.dc));
  act_.clear();
  blocks_.clear();
  act_.push_back(s.bytes((size_t)B_ * 16 * cpad(c0) * 2));
  in_.assign(1, act_[0]);
  int res = 4;
  for (int i = 0; i < a.n_g; ++i) {
    GBlock g;
    g.B = B_; g.H = res; g.W = res; g.cin = a.g_mult[i] * a.ch; g.cout = a.g_mult[i + 1] * a.ch;
    g.dc = a.dc; g.npi = a.npi; g.f32 = false; g.bn_eps = a.bn_eps; g.sn_eps = a.sn_eps;
    g.keep_dgrad = true;
    g.plan_saved(s);
    blocks_.push_back(g);
    res *= 2;
    act_.push_back(s.bytes((size_t)B_ * res * res * cpad(g.cout) * 2));
    if (res == a.attn_res) {
      attn_after_ = i;
      attn_.B = B_; attn_.H = res; attn_.W = res; attn_.C = g.cout; attn_.npi = a.npi; attn_.sn_eps = a.sn_eps;
      attn_.plan_saved(s);
      attn_out_ = s.bytes((size_t)B_ * res * res * cpad(g.cout) * 2);
    }
    in_.push_back(i == attn_after_ ? attn_out_ : act_[i + 1]);
  }
  head_.B = B_; head_.H = a.img; head_.W = a.img; head_.C = a.g_mult[a.n_g] * a.ch;
  head_.npi = a.npi; head_.bn_eps = a.bn_eps; head_.sn_eps = a.sn_eps;
  head_.plan_saved(s);
}

struct GNetWs {
  void *g0, *g1;       // ping-pong activation gradients (bf16)
  float *dlin, *dcond, *part;
  void* head;          // output layer workspace
  size_t head_bytes;
  void* blk;           // block workspace
  size_t blk_bytes;
};

static GNetWs gnet_carve(const Arch& a, int B, const std::vector<GBlock>& blocks, const Attn* attn, Arena& w,
                         int n_cu) {
  GNetWs r;
  size_t maxact = (size_t)B * 16 * cpad(a.g_mult[0] * a.ch);
  int res = 4;
  size_t blk = 0;
  for (const GBlock& g : blocks) {
    res *= 2;
    maxact = std::max(maxact, (size_t)B * res * res * std::max(cpad(g.cin), cpad(g.cout)));
    blk = std::max(blk, g.ws_size(n_cu));
  }
  if (attn) blk = std::max(blk, attn->ws_size(n_cu));
  const int c0 = a.g_mult[0] * a.ch;
  blk = std::max(blk, sn_ws_bytes(16LL * c0, a.zc));
  r.g0 = w.bytes(maxact * 2);
  r.g1 = w.bytes(maxact * 2);
  r.dlin = w.f32(16LL * c0 * a.zc);
  r.dcond = w.f32((size_t)B * a.dc);
  r.part = w.f32(kSnbParts);
  GOut head;
  head.B = B; head.H = a.img; head.W = a.img; head.C = a.g_mult[a.n_g] * a.ch;
  r.head_bytes = head.ws_size();
  r.head = w.bytes(r.head_bytes);
  r.blk_bytes = blk;
  r.blk = w.bytes(blk);
  return r;
}

size_t GNet::ws_size(int n_cu) {
  Arena w(nullptr);
  gnet_carve(a_, B_, blocks_, attn_after_ >= 0 ? &attn_ : nullptr, w, n_cu);
  return w.off;
}

// Every SN weight of the network through one group of launches per power
// iteration phase (kSnGroupMax weights a launch), then every weight pack
// through one group of launches: the same kernels, per weight, as each
// module's own prep, so the results are identical, in a few launches
// instead of four per module.
void GNet::prep(hipStream_t st, const Params& P, void* sn_ws, bool for_bwd, bool pack) {
  const Arch& a = a_;
  std::vector<SnJob> sj;
  std::vector<PackJob> pk;
  sj.push_back(sn_job(P, "linear.w", lin_));
  for (int i = 0; i < a.n_g; ++i) blocks_[i].sn_jobs(sub(P, "g" + std::to_string(i) + "."), sj);
  if (attn_after_ >= 0) attn_.sn_jobs(sub(P, "attn."), sj);
  sj.push_back(sn_job(P, "out_conv.w", head_.sn_slot()));
  sn_power_iter_all(st, sj.data(), (int)sj.size(), a.npi, a.sn_eps, sn_ws);
  for (int i = 0; i < a.n_g; ++i) {
    if (pack) blocks_[i].pack_jobs(sub(P, "g" + std::to_string(i) + "."), for_bwd, pk);
    blocks_[i].prepped = true;
  }
  // (the attention packs divide by sigma, so they are redone after every
  // SN update, and after the SN launches above)
  if (attn_after_ >= 0) {
    attn_.pack_jobs(sub(P, "attn."), pk);
    attn_.prepped = true;
  }
  pack_all(st, false, pk.data(), (int)pk.size());
  head_.prepped = true;
  prepped_ = true;
}

void GNet::fwd(const Exec& ex, const Params& P, const float* z, const int32_t* y, float* img, bool for_bwd) {
  const Arch& a = a_;
  Arena w(ex.ws);
  GNetWs r = gnet_carve(a, B_, blocks_, attn_after_ >= 0 ? &attn_ : nullptr, w, ex.n_cu);
  Exec eb{ex.st, ex.n_cu, r.blk, r.blk_bytes};
  const int c0 = a.g_mult[0] * a.ch;
  if (!prepped_) sn_forward(eb, P, "linear.w", lin_, a.npi, a.sn_eps);
  glin_fwd(ex.st, z, a.dz, a.zc, P.w("linear.w"), lin_.sigma, P.w("linear.b"), B_, c0, (int)cpad(c0), act_[0]);
  const void* h = act_[0];
  for (int i = 0; i < a.n_g; ++i) {
    make_cond(ex.st, P.w("shared"), a.sd, y, z, a.dz, a.zc * (i + 1), a.zc, B_, cond_[i]);
    blocks_[i].fwd(eb, sub(P, "g" + std::to_string(i) + "."), h, cond_[i], act_[i + 1]);
    h = act_[i + 1];
    if (i == attn_after_) {
      attn_.fwd(eb, sub(P, "attn."), h, attn_out_, for_bwd);
      h = attn_out_;
    }
  }
  head_.fwd(Exec{ex.st, ex.n_cu, r.head, r.head_bytes}, P, h, img);
  img_ = img;
  // a later forward runs its own SN and packing unless prepped again
  for (GBlock& g : blocks_) g.prepped = false;
  attn_.prepped = head_.prepped = prepped_ = false;
}

void GNet::bwd(const Exec& ex, const Params& P, const float* z, const int32_t* y, const float* dimg, int ldd) {
  const Arch& a = a_;
  Arena w(ex.ws);
  GNetWs r = gnet_carve(a, B_, blocks_, attn_after_ >= 0 ? &attn_ : nullptr, w, ex.n_cu);
  Exec eb{ex.st, ex.n_cu, r.blk, r.blk_bytes, ex.side, ex.ev_fork, ex.ev_join};
  void* gcur = r.g0;
  void* gnext = r.g1;
  head_.bwd(Exec{ex.st, ex.n_cu, r.head, r.head_bytes}, P, in_[a.n_g], img_, dimg, ldd, gcur);
  for (int i = a.n_g - 1; i >= 0; --i) {
    if (i == attn_after_) {
      attn_.bwd(eb, sub(P, "attn."), act_[i + 1], gcur, gnext);
      std::swap(gcur, gnext);
    }
    blocks_[i].bwd(eb, sub(P, "g" + std::to_string(i) + "."), in_[i], cond_[i], gcur, gnext, r.dcond,
                   i != a.n_g - 1);
    std::swap(gcur, gnext);
  }
  const int c0 = a.g_mult[0] * a.ch;
  glin_bwd(ex.st, gcur, z, a.dz, a.zc, B_, c0, (int)cpad(c0), r.dlin, P.gr("linear.b"));
  sn_bwd(ex.st, r.dlin, P.w("linear.w"), lin_.u, lin_.v, lin_.sigma, 16 * c0, a.zc, 1, a.zc, nullptr,
         P.gr("linear.w"), r.part);
  shared_grad(ex.st, r.dcond, a.dc, y, B_, a.n_classes, a.sd, P.gr("shared"));
}

// ============================================================ G output layer
Layout gout_layout(int C) {
  Layout L;
  L.add("out_bn.gain", {C}, false);
  L.add("out_bn.bias", {C}, false);
  L.add("out_conv.w", {3, 3, 3, C}, true);
  L.add("out_conv.b", {3}, false);
  return L;
}

void GOut::plan_saved(Arena& s) {
  const int cp = (int)cpad(C);
  mean_ = s.f32(cp); rstd_ = s.f32(cp); gain_ = s.f32(cp); bias_ = s.f32(cp); scale_ = s.f32(cp);
  plan_slot(s, sn_, 3, 27LL * C);
}

struct GOutWs {
  float *da, *dw, *part;
  void* red;           // reductions, the SN iteration and the weight-gradient partials, in turn
  size_t red_bytes;
};

static GOutWs gout_carve(const GOut& g, Arena& w) {
  const int64_t M = (int64_t)g.B * g.H * g.W;
  GOutWs r;
  r.da = w.f32((size_t)M * cpad(g.C));
  r.dw = w.f32(27LL * g.C);
  r.part = w.f32(kSnbParts);
  r.red_bytes = std::max({ghead_ws_bytes(g.B, g.H, g.W, g.C), bn_bwd_ws_bytes(g.B, g.H * g.W, g.C),
                          bn_stats_ws_bytes(M, g.C), sn_ws_bytes(3, 27LL * g.C)});
  r.red = w.bytes(r.red_bytes);
  return r;
}

size_t GOut::ws_size() const {
  Arena w(nullptr);
  gout_carve(*this, w);
  return w.off;
}

void GOut::fwd(const Exec& ex, const Params& P, const void* x, float* img) {
  Arena w(ex.ws);
  const GOutWs r = gout_carve(*this, w);
  PG_CHECK(w.off <= ex.ws_bytes, "output layer: workspace too small");
  const int cp = (int)cpad(C);
  bn_stats(ex.st, false, x, (int64_t)B * H * W, C, cp, bn_eps, mean_, rstd_, r.red);
  cbn_tables(ex.st, nullptr, 0, nullptr, nullptr, nullptr, nullptr, P.w("out_bn.gain"), P.w("out_bn.bias"), rstd_,
             1, C, cp, gain_, bias_, scale_);
  if (!prepped) sn_forward(Exec{ex.st, ex.n_cu, r.red, r.red_bytes}, P, "out_conv.w", sn_, npi, sn_eps);
  ghead_fwd(ex.st, x, B, H, W, C, cp, mean_, scale_, bias_, P.w("out_conv.w"), sn_.sigma, P.w("out_conv.b"), img);
}

void GOut::bwd(const Exec& ex, const Params& P, const void* x, const float* img, const float* dimg, int ldd,
               void* dx) {
  Arena w(ex.ws);
  const GOutWs r = gout_carve(*this, w);
  PG_CHECK(w.off <= ex.ws_bytes, "output layer: workspace too small");
  const int cp = (int)cpad(C);
  ghead_bwd(ex.st, dimg, ldd, img, x, B, H, W, C, cp, mean_, scale_, bias_, P.w("out_conv.w"), sn_.sigma, r.da,
            r.dw, P.gr("out_conv.b"), r.red);
  sn_bwd(ex.st, r.dw, P.w("out_conv.w"), sn_.u, sn_.v, sn_.sigma, 3, C, 3, C, nullptr, P.gr("out_conv.w"), r.part);
  bn_bwd(ex.st, false, r.da, false, x, B, H, W, C, cp, mean_, rstd_, gain_, bias_, 0, nullptr, dx,
         P.gr("out_bn.gain"), P.gr("out_bn.bias"), 0, r.red);
}

// =================================================================== D
void DNet::plan_saved(Arena& s) {
  const Arch& a = a_;
  act_.clear();
  blocks_.clear();
  act_.push_back(s.bytes((size_t)N_ * a.img * a.img * 32 * 2));
  in_.assign(1, act_[0]);
  const auto specs = d_specs(a);
  for (int j = 0; j < (int)specs.size(); ++j) {
    const DSpec& sp = specs[j];
    DBlock b;
    b.B = N_; b.H = sp.H; b.W = sp.W; b.cin = sp.cin; b.cout = sp.cout; b.npi = a.npi;
    b.preact = sp.preact; b.down = sp.down; b.lsc = sp.lsc; b.f32 = false; b.sn_eps = a.sn_eps;
    b.im2col = j == 0;   // the image enters as 3x3 patches
    b.keep_dgrad = true;
    b.plan_saved(s);
    blocks_.push_back(b);
    act_.push_back(s.bytes((size_t)N_ * b.Ho * b.Wo * cpad(sp.cout) * 2));
    if (sp.attn) {
      attn_after_ = j;
      attn_.B = N_; attn_.H = b.Ho; attn_.W = b.Wo; attn_.C = sp.cout; attn_.npi = a.npi; attn_.sn_eps = a.sn_eps;
      attn_.plan_saved(s);
      attn_out_ = s.bytes((size_t)N_ * b.Ho * b.Wo * cpad(sp.cout) * 2);
    }
    in_.push_back(j == attn_after_ ? attn_out_ : act_[j + 1]);
  }
  const int c = a.d_mult[a.n_d - 1] * a.ch;
  hs_ = s.f32((size_t)N_ * c);
  plan_slot(s, head_, 1, c);
  plan_slot(s, emb_, a.n_classes, c);
}

struct DNetWs {
  void *g0, *g1;
  float *dw, *dE, *part;
  void* blk;
  size_t blk_bytes;
};

static DNetWs dnet_carve(const Arch& a, int N, const std::vector<DBlock>& blocks, const Attn* attn, Arena& w,
                         int n_cu) {
  DNetWs r;
  size_t maxact = 0, blk = 0;
  for (const DBlock& b : blocks) {
    maxact = std::max(maxact, (size_t)N * b.H * b.W * std::max(cpad(b.cin), cpad(b.cout)));
    blk = std::max(blk, b.ws_size(n_cu));
  }
  if (attn) blk = std::max(blk, attn->ws_size(n_cu));
  const int c = a.d_mult[a.n_d - 1] * a.ch;
  blk = std::max({blk, sn_ws_bytes(1, c), sn_ws_bytes(a.n_classes, c)});
  r.g0 = w.bytes(maxact * 2);
  r.g1 = w.bytes(maxact * 2);
  r.dw = w.f32(c);
  r.dE = w.f32((size_t)a.n_classes * c);
  r.part = w.f32(kSnbParts);
  r.blk_bytes = blk;
  r.blk = w.bytes(blk);
  return r;
}

size_t DNet::ws_size(int n_cu) {
  Arena w(nullptr);
  dnet_carve(a_, N_, blocks_, attn_after_ >= 0 ? &attn_ : nullptr, w, n_cu);
  return w.off;
}

void DNet::prep(hipStream_t st, const Params& P, void* sn_ws, bool for_bwd) {
  const Arch& a = a_;
  std::vector<SnJob> sj;
  std::vector<PackJob> pk;
  for (int j = 0; j < (int)blocks_.size(); ++j) blocks_[j].sn_jobs(sub(P, "d" + std::to_string(j) + "."), sj);
  if (attn_after_ >= 0) attn_.sn_jobs(sub(P, "attn."), sj);
  sj.push_back(sn_job(P, "head.w", head_));
  sj.push_back(sn_job(P, "embed", emb_));
  sn_power_iter_all(st, sj.data(), (int)sj.size(), a.npi, a.sn_eps, sn_ws);
  for (int j = 0; j < (int)blocks_.size(); ++j) {
    blocks_[j].pack_jobs(sub(P, "d" + std::to_string(j) + "."), for_bwd, pk);
    blocks_[j].prepped = true;
  }
  if (attn_after_ >= 0) {
    attn_.pack_jobs(sub(P, "attn."), pk);
    attn_.prepped = true;
  }
  pack_all(st, false, pk.data(), (int)pk.size());
  prepped_ = true;
}

void DNet::fwd(const Exec& ex, const Params& P, const float* x, const int32_t* y, float* out) {
  const Arch& a = a_;
  Arena w(ex.ws);
  DNetWs r = dnet_carve(a, N_, blocks_, attn_after_ >= 0 ? &attn_ : nullptr, w, ex.n_cu);
  Exec eb{ex.st, ex.n_cu, r.blk, r.blk_bytes};
  img_to_im2col(ex.st, x, N_, a.img, a.img, act_[0]);
  const void* h = act_[0];
  for (int j = 0; j < (int)blocks_.size(); ++j) {
    blocks_[j].fwd(eb, sub(P, "d" + std::to_string(j) + "."), h, act_[j + 1]);
    h = act_[j + 1];
    if (j == attn_after_) {
      attn_.fwd(eb, sub(P, "attn."), h, attn_out_);
      h = attn_out_;
    }
  }
  const DBlock& last = blocks_.back();
  if (!prepped_) {
    sn_forward(eb, P, "head.w", head_, a.npi, a.sn_eps);
    sn_forward(eb, P, "embed", emb_, a.npi, a.sn_eps);
  }
  for (DBlock& b : blocks_) b.prepped = false;
  attn_.prepped = prepped_ = false;
  dhead_fwd(ex.st, h, N_, last.Ho * last.Wo, last.cout, last.Cop, y, P.w("head.w"), head_.sigma, P.w("head.b"),
            P.w("embed"), emb_.sigma, hs_, out);
}

void DNet::bwd(const Exec& ex, const Params& P, const int32_t* y, const float* dout, float* dimg, bool wgrad) {
  const Arch& a = a_;
  Arena w(ex.ws);
  DNetWs r = dnet_carve(a, N_, blocks_, attn_after_ >= 0 ? &attn_ : nullptr, w, ex.n_cu);
  Exec eb{ex.st, ex.n_cu, r.blk, r.blk_bytes, ex.side, ex.ev_fork, ex.ev_join};
  const DBlock& last = blocks_.back();
  const int nb = (int)blocks_.size();
  const void* xl = in_[nb];
  void* gcur = r.g0;
  void* gnext = r.g1;
  dhead_bwd(ex.st, xl, N_, last.Ho * last.Wo, last.cout, last.Cop, y, dout, hs_, P.w("head.w"), head_.sigma,
            P.w("embed"), emb_.sigma, a.n_classes, gcur, wgrad ? r.dw : nullptr, P.gr("head.b"), r.dE);
  if (wgrad) {
    sn_bwd(ex.st, r.dw, P.w("head.w"), head_.u, head_.v, head_.sigma, 1, last.cout, 1, last.cout, nullptr,
           P.gr("head.w"), r.part);
    sn_bwd(ex.st, r.dE, P.w("embed"), emb_.u, emb_.v, emb_.sigma, a.n_classes, last.cout, 1, last.cout, nullptr,
           P.gr("embed"), r.part);
  }
  for (int j = nb - 1; j >= 0; --j) {
    if (j == attn_after_) {
      attn_.bwd(eb, sub(P, "attn."), act_[j + 1], gcur, gnext, wgrad);
      std::swap(gcur, gnext);
    }
    void* dx = j > 0 ? gnext : (void*)dimg;
    blocks_[j].bwd(eb, sub(P, "d" + std::to_string(j) + "."), in_[j], gcur, dx, j == 0, wgrad);
    std::swap(gcur, gnext);
  }
}

// =================================================================== step
struct StepWs {
  void* gsaved;
  void* dsaved;
  float *ximg, *logits, *dout, *dimg, *dloss;
  int32_t* ylab;
  void* net;
  size_t net_bytes;
  void* side;          // SN workspace of the second stream's weight preparation
};

static StepWs step_carve(const Arch& a, int B, Arena& w, GNet& g, DNet& d2, DNet& d1, int n_cu) {
  StepWs r;
  Arena gs(w.base ? w.base + w.off : nullptr);
  g.plan_saved(gs);
  r.gsaved = w.bytes(gs.off);
  Arena ds2(w.base ? w.base + w.off : nullptr), ds1(w.base ? w.base + w.off : nullptr);
  d2.plan_saved(ds2);
  d1.plan_saved(ds1);
  r.dsaved = w.bytes(std::max(ds2.off, ds1.off));
  const int64_t pix = (int64_t)a.img * a.img;
  r.ximg = w.f32((size_t)2 * B * pix * 3);
  r.ylab = (int32_t*)w.bytes((size_t)2 * B * 4);
  r.logits = w.f32(2 * B);
  r.dout = w.f32(2 * B);
  r.dimg = w.f32((size_t)B * pix * 4);
  r.dloss = w.f32(64);
  r.net_bytes = std::max({g.ws_size(n_cu), d2.ws_size(n_cu), d1.ws_size(n_cu)});
  r.net = w.bytes(r.net_bytes);
  r.side = w.bytes(std::max(sn_ws_all(g_layout(a)), sn_ws_all(d_layout(a))));
  return r;
}

size_t train_step_ws(const paragan_biggan_desc* d, int n_cu) {
  const Arch a = arch_from(d);
  GNet g(a, d->B);
  DNet d2(a, 2 * d->B), d1(a, d->B);
  Arena w(nullptr);
  step_carve(a, d->B, w, g, d2, d1, n_cu);
  return w.off;
}

namespace {
// The pieces of a training iteration over one workspace: the generator
// (batch B), the discriminator on the 2B batch of a D step and on the B
// images of a G step (their saved buffers share one region).
struct StepRun {
  Arch a;
  int B;
  hipStream_t st;
  GNet g;
  DNet d2, d1;
  StepWs r;
  Exec ex;
  Layout LG, LD;
  Params PG, PD;
  int64_t pix;
  StepRun(paragan_ctx* ctx, const paragan_biggan_desc* d, paragan_net_state* G, paragan_net_state* D, void* ws)
      : a(arch_from(d)), B(d->B), st(ctx->stream), g(a, B), d2(a, 2 * B), d1(a, B) {
    Arena w(ws);
    r = step_carve(a, B, w, g, d2, d1, ctx->n_cu);
    ex = Exec{st, ctx->n_cu, r.net, r.net_bytes};
    if (ctx->overlap_wgrad) {
      if (!ctx->wside) {
        PG_HIP(hipStreamCreateWithFlags(&ctx->wside, hipStreamNonBlocking));
        for (hipEvent_t& e : ctx->wev) PG_HIP(hipEventCreateWithFlags(&e, hipEventDisableTiming));
      }
      ex.side = ctx->wside;
      ex.ev_fork = ctx->wev[0];
      ex.ev_join = ctx->wev[1];
    }
    LG = g_layout(a);
    LD = d_layout(a);
    PG = Params{&LG, "", G ? G->params : nullptr, G ? G->u : nullptr, G ? G->grads : nullptr};
    PD = Params{&LD, "", D ? D->params : nullptr, D ? D->u : nullptr, D ? D->grads : nullptr};
    pix = (int64_t)a.img * a.img;
  }
  static void optimise(hipStream_t st, const paragan_optim& o, paragan_net_state* N, int64_t n) {
    N->opt_t += 1;
    optim_step(st, o.kind, N->params, N->grads, N->opt_m, N->opt_v, n, o.beta1, o.beta2, o.lr, o.eps, N->opt_t);
  }
  // D step on the batch already in r.ximg / r.ylab: forward, hinge (L_D to
  // *loss), backward with weight gradients, D's optimiser
  void d_update(const paragan_biggan_desc* d, paragan_net_state* D, float* loss) {
    d2.fwd(ex, PD, r.ximg, r.ylab, r.logits);
    hinge(st, r.logits, B, B, false, r.dout, loss);
    d2.bwd(ex, PD, r.ylab, r.dout, nullptr, true);
    optimise(st, d->opt_d, D, LD.n_params);
  }
  void stage_real(const float* x_real, const int32_t* y_real, const int32_t* y_fake) {
    PG_HIP(hipMemcpyAsync(r.ximg, x_real, (size_t)B * pix * 3 * 4, hipMemcpyDeviceToDevice, st));
    PG_HIP(hipMemcpyAsync(r.ylab, y_real, (size_t)B * 4, hipMemcpyDeviceToDevice, st));
    PG_HIP(hipMemcpyAsync(r.ylab + B, y_fake, (size_t)B * 4, hipMemcpyDeviceToDevice, st));
  }
  float* fake_half() { return r.ximg + (size_t)B * pix * 3; }
  // G step: G forward, D forward (u updated), hinge (L_G to *loss), D input
  // gradient, G backward, G's optimiser
  // (between_fwds runs after G's forward, before D's: the point where the
  // fused step waits for D's preparation)
  template <typename F>
  void g_update(const paragan_biggan_desc* d, paragan_net_state* G, const float* z, const int32_t* y,
                float* loss, F&& between_fwds) {
    g.fwd(ex, PG, z, y, r.ximg);
    between_fwds();
    d1.fwd(ex, PD, r.ximg, y, r.logits);
    hinge(st, r.logits, 0, B, true, r.dout, loss);
    d1.bwd(ex, PD, y, r.dout, r.dimg, false);
    g.bwd(ex, PG, z, y, r.dimg, 4);
    optimise(st, d->opt_g, G, LG.n_params);
  }
  void losses_to_host(float* host, int n) {
    PG_HIP(hipMemcpyAsync(host, r.dloss, (size_t)n * 4, hipMemcpyDeviceToHost, st));
    PG_HIP(hipStreamSynchronize(st));
  }
};
}  // namespace

void g_sample(paragan_ctx* ctx, const paragan_biggan_desc* d, paragan_net_state* G, const float* z,
              const int32_t* y, float* img, void* ws) {
  StepRun R(ctx, d, G, nullptr, ws);
  R.g.fwd(R.ex, R.PG, z, y, img, false);
}

void d_step(paragan_ctx* ctx, const paragan_biggan_desc* d, paragan_net_state* D, const float* x_real,
            const int32_t* y_real, const float* x_fake, const int32_t* y_fake, void* ws, float* loss_host) {
  StepRun R(ctx, d, nullptr, D, ws);
  R.stage_real(x_real, y_real, y_fake);
  PG_HIP(hipMemcpyAsync(R.fake_half(), x_fake, (size_t)R.B * R.pix * 3 * 4, hipMemcpyDeviceToDevice, R.st));
  R.d_update(d, D, R.r.dloss);
  R.losses_to_host(loss_host, 1);
}

void g_step(paragan_ctx* ctx, const paragan_biggan_desc* d, paragan_net_state* G, paragan_net_state* D,
            const float* z, const int32_t* y, void* ws, float* loss_host) {
  StepRun R(ctx, d, G, D, ws);
  R.g_update(d, G, z, y, R.r.dloss, [] {});
  R.losses_to_host(loss_host, 1);
}

void train_step(paragan_ctx* ctx, const paragan_biggan_desc* d, paragan_net_state* G, paragan_net_state* D,
                const paragan_step_inputs* in, int n_D, void* ws, float* losses_host) {
  StepRun R(ctx, d, G, D, ws);
  hipStream_t st = R.st;
  // The forwards' SN power iterations and weight packing (which read only
  // parameters) run on a second stream, each network's ahead of its forward
  // and behind the work that last used its SN state or changed its
  // parameters: D's behind the previous optimiser step (overlapping G's
  // forward), G's behind the previous G forward (overlapping D's forward and
  // backward).  G's parameters do not change before the G step's optimiser,
  // so its weights are packed once per step (forward and data-gradient
  // packs), and its later preparations run only the SN power iterations.
  // The G step waits for D's preparation only after G's forward.  The
  // kernels are the same as on the one-stream path, so the results are too.
  if (!ctx->side) {
    PG_HIP(hipStreamCreateWithFlags(&ctx->side, hipStreamNonBlocking));
    for (hipEvent_t& e : ctx->ev) PG_HIP(hipEventCreateWithFlags(&e, hipEventDisableTiming));
  }
  hipStream_t sd = ctx->side;
  try {
    hipEvent_t ev_main = ctx->ev[0], ev_main2 = ctx->ev[1], ev_g = ctx->ev[2], ev_d = ctx->ev[3];
    auto side_after_main = [&](hipEvent_t e) {
      PG_HIP(hipEventRecord(e, st));
      PG_HIP(hipStreamWaitEvent(sd, e, 0));
    };
    auto main_after = [&](hipEvent_t e) { PG_HIP(hipStreamWaitEvent(st, e, 0)); };
    side_after_main(ev_main2);
    R.g.prep(sd, R.PG, R.r.side, true);
    PG_HIP(hipEventRecord(ev_g, sd));
    for (int k = 0; k < n_D; ++k) {
      side_after_main(ev_main);
      R.d2.prep(sd, R.PD, R.r.side, true);
      PG_HIP(hipEventRecord(ev_d, sd));
      R.stage_real(in->x_real[k], in->y_real[k], in->y_fake[k]);
      main_after(ev_g);
      R.g.fwd(R.ex, R.PG, in->z_fake[k], in->y_fake[k], R.fake_half(), false);
      side_after_main(ev_main2);
      R.g.prep(sd, R.PG, R.r.side, false, false);   // SN for the next D step's or the G step's forward
      PG_HIP(hipEventRecord(ev_g, sd));
      main_after(ev_d);
      R.d_update(d, D, R.r.dloss + k);
    }
    side_after_main(ev_main);
    R.d1.prep(sd, R.PD, R.r.side, true);
    PG_HIP(hipEventRecord(ev_d, sd));
    main_after(ev_g);
    R.g_update(d, G, in->z_g, in->y_g, R.r.dloss + n_D, [&] { main_after(ev_d); });
    R.losses_to_host(losses_host, n_D + 1);
  } catch (...) {
    // leave neither stream running on the caller's buffers
    (void)hipStreamSynchronize(sd);
    (void)hipStreamSynchronize(st);
    throw;
  }
}

// =================================================================== async
// The asynchronous update scheme (Numerical Optimizations, "Asynchronous
// Update Scheme"): within one iteration the generator step runs against a
// snapshot of the discriminator taken at the iteration's start, on the
// context's second stream, while the n_D discriminator steps run on the
// caller's stream on the previous iteration's generator samples (img_buff,
// one iteration stale).  The two sides share no state until the join at the
// end, where this iteration's samples replace img_buff.
struct AsyncWs {
  void *gsaved, *ssaved, *dsaved;     // G (batch n_D B), the snapshot D (n_D B), the stepping D (2B)
  float *snap_p, *snap_u;             // the snapshot's parameters and SN vectors
  float *gimg, *glog, *gdout, *gdimg, *gloss;
  float *dimg, *dlog, *ddout, *dloss;
  int32_t* dlab;
  void *gnet, *dnet;
  size_t gnet_bytes, dnet_bytes;
};

template <typename Net>
static void* carve_saved(Arena& w, Net& net) {
  Arena s(w.base ? w.base + w.off : nullptr);
  net.plan_saved(s);
  return w.bytes(s.off);
}

static AsyncWs async_carve(const Arch& a, int B, int n_D, Arena& w, GNet& g, DNet& ds, DNet& d2, int n_cu) {
  AsyncWs r;
  const int BG = n_D * B;
  const int64_t pix = (int64_t)a.img * a.img;
  r.gsaved = carve_saved(w, g);
  r.ssaved = carve_saved(w, ds);
  r.dsaved = carve_saved(w, d2);
  const Layout LD = d_layout(a);
  r.snap_p = w.f32(LD.n_params);
  r.snap_u = w.f32(std::max<int64_t>(LD.n_u, 1));
  r.gimg = w.f32((size_t)BG * pix * 3);
  r.glog = w.f32(BG);
  r.gdout = w.f32(BG);
  r.gdimg = w.f32((size_t)BG * pix * 4);
  r.gloss = w.f32(64);
  r.dimg = w.f32((size_t)2 * B * pix * 3);
  r.dlab = (int32_t*)w.bytes((size_t)2 * B * 4);
  r.dlog = w.f32(2 * B);
  r.ddout = w.f32(2 * B);
  r.dloss = w.f32(64);
  r.gnet_bytes = std::max(g.ws_size(n_cu), ds.ws_size(n_cu));
  r.gnet = w.bytes(r.gnet_bytes);
  r.dnet_bytes = d2.ws_size(n_cu);
  r.dnet = w.bytes(r.dnet_bytes);
  return r;
}

size_t async_step_ws(const paragan_biggan_desc* d, int n_D, int n_cu) {
  const Arch a = arch_from(d);
  GNet g(a, n_D * d->B);
  DNet ds(a, n_D * d->B), d2(a, 2 * d->B);
  Arena w(nullptr);
  async_carve(a, d->B, n_D, w, g, ds, d2, n_cu);
  return w.off;
}

void async_step(paragan_ctx* ctx, const paragan_biggan_desc* d, paragan_net_state* G, paragan_net_state* D,
                const paragan_async_inputs* in, int n_D, void* ws, float* losses_host) {
  const Arch a = arch_from(d);
  const int B = d->B, BG = n_D * B;
  GNet g(a, BG);
  DNet ds(a, BG), d2(a, 2 * B);
  Arena w(ws);
  const AsyncWs r = async_carve(a, B, n_D, w, g, ds, d2, ctx->n_cu);
  hipStream_t st = ctx->stream;
  if (!ctx->side) {
    PG_HIP(hipStreamCreateWithFlags(&ctx->side, hipStreamNonBlocking));
    for (hipEvent_t& e : ctx->ev) PG_HIP(hipEventCreateWithFlags(&e, hipEventDisableTiming));
  }
  hipStream_t sg = ctx->side;
  const Layout LG = g_layout(a), LD = d_layout(a);
  const Params PG{&LG, "", G->params, G->u, G->grads};
  const Params PD{&LD, "", D->params, D->u, D->grads};
  const Params PS{&LD, "", r.snap_p, r.snap_u, nullptr};
  const int64_t pix = (int64_t)a.img * a.img;
  try {
    // the snapshot of D at the start of the iteration
    PG_HIP(hipMemcpyAsync(r.snap_p, D->params, (size_t)LD.n_params * 4, hipMemcpyDeviceToDevice, st));
    PG_HIP(hipMemcpyAsync(r.snap_u, D->u, (size_t)LD.n_u * 4, hipMemcpyDeviceToDevice, st));
    PG_HIP(hipEventRecord(ctx->ev[0], st));
    PG_HIP(hipStreamWaitEvent(sg, ctx->ev[0], 0));
    // generator side: samples, the snapshot's predictions (pred_buff),
    // L_G, the input gradient through the snapshot, G's backward and step
    const Exec eg{sg, ctx->n_cu, r.gnet, r.gnet_bytes};
    g.fwd(eg, PG, in->z, in->y, r.gimg);
    ds.fwd(eg, PS, r.gimg, in->y, r.glog);
    hinge(sg, r.glog, 0, BG, true, r.gdout, r.gloss);
    ds.bwd(eg, PS, in->y, r.gdout, r.gdimg, false);
    g.bwd(eg, PG, in->z, in->y, r.gdimg, 4);
    G->opt_t += 1;
    optim_step(sg, d->opt_g.kind, G->params, G->grads, G->opt_m, G->opt_v, LG.n_params, d->opt_g.beta1,
               d->opt_g.beta2, d->opt_g.lr, d->opt_g.eps, G->opt_t);
    PG_HIP(hipEventRecord(ctx->ev[1], sg));
    // discriminator side: step k on B real images and the k-th B of the
    // previous iteration's samples
    const Exec ed{st, ctx->n_cu, r.dnet, r.dnet_bytes};
    for (int k = 0; k < n_D; ++k) {
      PG_HIP(hipMemcpyAsync(r.dimg, in->x_real[k], (size_t)B * pix * 3 * 4, hipMemcpyDeviceToDevice, st));
      PG_HIP(hipMemcpyAsync(r.dimg + (size_t)B * pix * 3, in->img_buff + (size_t)k * B * pix * 3,
                            (size_t)B * pix * 3 * 4, hipMemcpyDeviceToDevice, st));
      PG_HIP(hipMemcpyAsync(r.dlab, in->y_real[k], (size_t)B * 4, hipMemcpyDeviceToDevice, st));
      PG_HIP(hipMemcpyAsync(r.dlab + B, in->lab_buff + (size_t)k * B, (size_t)B * 4, hipMemcpyDeviceToDevice, st));
      d2.fwd(ed, PD, r.dimg, r.dlab, r.dlog);
      hinge(st, r.dlog, B, B, false, r.ddout, r.dloss + k);
      d2.bwd(ed, PD, r.dlab, r.ddout, nullptr, true);
      D->opt_t += 1;
      optim_step(st, d->opt_d.kind, D->params, D->grads, D->opt_m, D->opt_v, LD.n_params, d->opt_d.beta1,
                 d->opt_d.beta2, d->opt_d.lr, d->opt_d.eps, D->opt_t);
    }
    // join, then this iteration's samples become the next one's img_buff
    PG_HIP(hipStreamWaitEvent(st, ctx->ev[1], 0));
    PG_HIP(hipMemcpyAsync(in->img_buff, r.gimg, (size_t)BG * pix * 3 * 4, hipMemcpyDeviceToDevice, st));
    PG_HIP(hipMemcpyAsync(in->lab_buff, in->y, (size_t)BG * 4, hipMemcpyDeviceToDevice, st));
    PG_HIP(hipMemcpyAsync(in->pred_buff, r.glog, (size_t)BG * 4, hipMemcpyDeviceToDevice, st));
    PG_HIP(hipMemcpyAsync(r.dloss + n_D, r.gloss, 4, hipMemcpyDeviceToDevice, st));
    PG_HIP(hipMemcpyAsync(losses_host, r.dloss, (size_t)(n_D + 1) * 4, hipMemcpyDeviceToHost, st));
    PG_HIP(hipStreamSynchronize(st));
  } catch (...) {
    (void)hipStreamSynchronize(sg);
    (void)hipStreamSynchronize(st);
    throw;
  }
}

}  // namespace pg
