// BigGAN networks and the G+D train step (host runtime).
#pragma once
#include "../../include/paragan.h"
#include "attn.hpp"
#include "blocks.hpp"
#include "heads.hpp"

namespace pg {

struct Arch {
  int img, ch, n_g, n_d, attn_res, n_classes, dz, sd, zc, dc;
  std::vector<int> g_mult, d_mult, d_down;
  int npi;
  float bn_eps, sn_eps;
};

Arch arch_from(const paragan_biggan_desc* d);
void check_arch(const paragan_biggan_desc* d);
Layout g_layout(const Arch& a);
Layout d_layout(const Arch& a);

struct DSpec {
  int cin, cout, H, W;
  bool preact, down, lsc, attn;
};
std::vector<DSpec> d_specs(const Arch& a);

// Generator output layer, fp32 arithmetic: BN with batch statistics and an
// affine gain / bias -> ReLU -> SN conv3x3 (C -> 3, bias) -> tanh.
// Parameters (named): out_bn.gain out_bn.bias out_conv.w out_conv.b.
class GOut {
 public:
  int B = 0, H = 0, W = 0, C = 0, npi = 1;
  float bn_eps = 1e-5f, sn_eps = 1e-12f;
  void plan_saved(Arena& s);
  size_t ws_size() const;
  // x: bf16 [B][H][W][cpad(C)]; img: fp32 [B][H][W][3]
  void fwd(const Exec& ex, const Params& P, const void* x, float* img);
  // prepped: the SN of out_conv.w already ran (GNet::prep, into sn_slot())
  bool prepped = false;
  SNSlot& sn_slot() { return sn_; }
  // img: this layer's forward output; dimg: fp32 [B][H][W][ldd];
  // dx: bf16 [B][H][W][cpad(C)]
  void bwd(const Exec& ex, const Params& P, const void* x, const float* img, const float* dimg, int ldd,
           void* dx);

 private:
  SNSlot sn_;
  float *mean_ = nullptr, *rstd_ = nullptr, *gain_ = nullptr, *bias_ = nullptr, *scale_ = nullptr;
};
Layout gout_layout(int C);

class GNet {
 public:
  GNet(const Arch& a, int B) : a_(a), B_(B) {}
  void plan_saved(Arena& s);
  size_t ws_size(int n_cu);
  // img: fp32 [B][img][img][3]
  // for_bwd = false: no backward will follow this forward
  // The forward's SN power iterations and weight packing of every layer on
  // stream st (sn_ws: sn_ws_all of the layout); the next fwd then skips them.
  // for_bwd: the blocks' data-gradient weights too, for the next bwd.
  // pack = false: the SN power iterations only, the packed weights of the
  // last packing prep being still those of the parameters (the packs hold
  // unnormalised weights; sigma enters in the conv epilogues)
  void prep(hipStream_t st, const Params& P, void* sn_ws, bool for_bwd = false, bool pack = true);
  void fwd(const Exec& ex, const Params& P, const float* z, const int32_t* y, float* img, bool for_bwd = true);
  // dimg: fp32 [B][img][img][ldd]
  void bwd(const Exec& ex, const Params& P, const float* z, const int32_t* y, const float* dimg, int ldd);

 private:
  Arch a_;
  bool prepped_ = false;
  int B_;
  std::vector<GBlock> blocks_;
  Attn attn_;
  int attn_after_ = -1;
  std::vector<void*> act_;     // act_[0]: linear output; act_[i+1]: output of block i
  std::vector<void*> in_;      // in_[i]: input of block i (attention output after the attention block)
  void* attn_out_ = nullptr;
  std::vector<float*> cond_;
  SNSlot lin_;
  GOut head_;
  float* img_ = nullptr;
};

class DNet {
 public:
  DNet(const Arch& a, int N) : a_(a), N_(N) {}
  void plan_saved(Arena& s);
  size_t ws_size(int n_cu);
  // x: fp32 images [N][img][img][3]; out: fp32 logits [N]
  void prep(hipStream_t st, const Params& P, void* sn_ws, bool for_bwd = false);   // as GNet::prep
  void fwd(const Exec& ex, const Params& P, const float* x, const int32_t* y, float* out);
  // wgrad = false: input gradient only (dimg fp32 [N][img][img][4], channels 0..2)
  void bwd(const Exec& ex, const Params& P, const int32_t* y, const float* dout, float* dimg, bool wgrad);

 private:
  Arch a_;
  bool prepped_ = false;
  int N_;
  std::vector<DBlock> blocks_;
  Attn attn_;
  int attn_after_ = -1;
  std::vector<void*> act_;     // act_[0]: bf16 image; act_[j+1]: output of block j
  std::vector<void*> in_;      // in_[j]: input of block j
  void* attn_out_ = nullptr;
  float* hs_ = nullptr;
  SNSlot head_, emb_;
};

size_t train_step_ws(const paragan_biggan_desc* d, int n_cu);
void g_sample(paragan_ctx* ctx, const paragan_biggan_desc* d, paragan_net_state* G, const float* z,
              const int32_t* y, float* img, void* ws);
void d_step(paragan_ctx* ctx, const paragan_biggan_desc* d, paragan_net_state* D, const float* x_real,
            const int32_t* y_real, const float* x_fake, const int32_t* y_fake, void* ws, float* loss_host);
void g_step(paragan_ctx* ctx, const paragan_biggan_desc* d, paragan_net_state* G, paragan_net_state* D,
            const float* z, const int32_t* y, void* ws, float* loss_host);
size_t async_step_ws(const paragan_biggan_desc* d, int n_D, int n_cu);
void async_step(paragan_ctx* ctx, const paragan_biggan_desc* d, paragan_net_state* G, paragan_net_state* D,
                const paragan_async_inputs* in, int n_D, void* ws, float* losses_host);
void train_step(paragan_ctx* ctx, const paragan_biggan_desc* d, paragan_net_state* G, paragan_net_state* D,
                const paragan_step_inputs* in, int n_D, void* ws, float* losses_host);

}  // namespace pg
