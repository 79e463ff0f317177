// Host runtime: parameter layouts, buffer planning, and the residual-block
// executors used by both the per-block C-ABI calls and the train step.
#pragma once
#include <string>
#include <vector>

#include "misc.hpp"

namespace pg {

// Sequential carving of a caller-owned buffer; with a null base it only
// measures (the *_sizes() queries run the same plan with base == nullptr).
struct Arena {
  char* base;
  size_t off = 0;
  explicit Arena(void* b) : base((char*)b) {}
  void* bytes(size_t n) {
    const size_t o = off;
    off = align256(off + n);
    return base ? (void*)(base + o) : nullptr;
  }
  float* f32(size_t n) { return (float*)bytes(n * 4); }
};

struct Entry {
  std::string name;
  std::vector<int64_t> shape;
  bool sn;
  int64_t offset = 0, u_offset = -1;
  int64_t numel() const {
    int64_t n = 1;
    for (auto s : shape) n *= s;
    return n;
  }
};

struct Layout {
  std::vector<Entry> e;
  int64_t n_params = 0, n_u = 0;
  void add(const std::string& name, std::vector<int64_t> shape, bool sn) {
    Entry x{name, shape, sn};
    x.offset = n_params;
    n_params += x.numel();
    if (sn) {
      x.u_offset = n_u;
      n_u += shape[0];
    }
    e.push_back(x);
  }
  const Entry& get(const std::string& name) const;
  void add_prefixed(const std::string& prefix, const Layout& sub);
};

Layout gblock_layout(int cin, int cout, int dc);
Layout dblock_layout(int cin, int cout, bool lsc);
Layout attn_layout(int c);

// Parameters of one module resolved against flat buffers.
struct Params {
  const Layout* L;
  std::string prefix;
  const float* p;     // flat params
  float* u;           // flat u
  float* g;           // flat grads (may be null)
  const float* w(const std::string& n) const { return p + L->get(prefix + n).offset; }
  float* uu(const std::string& n) const { return u + L->get(prefix + n).u_offset; }
  float* gr(const std::string& n) const { return g + L->get(prefix + n).offset; }
  const Entry& ent(const std::string& n) const { return L->get(prefix + n); }
};

// One spectrally normalised weight: u, v and sigma of the last forward.
struct SNSlot {
  float* u = nullptr;
  float* v = nullptr;
  float* sigma = nullptr;
};

struct Exec {
  hipStream_t st;
  int n_cu;
  void* ws;           // scratch shared by the steps of one block call
  size_t ws_bytes;
  // with side set, a block backward runs its weight gradients there, beside
  // its data gradients on st, ordered by the two events (fork: st -> side,
  // join: side -> st); both streams are joined when the call returns
  hipStream_t side = nullptr;
  hipEvent_t ev_fork = nullptr, ev_join = nullptr;
};

// ----------------------------------------------------------- G block
struct GBlock {
  int B, H, W, cin, cout, dc, npi;
  bool f32;
  float bn_eps, sn_eps;
  int Cip, Cop;
  // saved by fwd for bwd
  SNSlot sn[7];
  void *wp1 = nullptr, *wp2 = nullptr, *wpsc = nullptr;
  float *mean1, *rstd1, *gain1, *bias1, *scale1;
  float *mean2, *rstd2, *gain2, *bias2, *scale2;
  void* h1 = nullptr;
  void *a1 = nullptr, *a2 = nullptr;   // relu(cbn1(x)), relu(cbn2(h1)): conv operands
  void plan_saved(Arena& a);
  size_t ws_size(int n_cu) const;
  // The forward's SN power iterations and weight packing: fwd runs them
  // itself unless prepped is set (then prep ran them before, e.g. on
  // another stream; sn_ws: sn_ws_all of the layout, or the block's share)
  bool prepped = false;
  // keep_dgrad (set before plan_saved): prep(for_bwd) also packs the
  // data-gradient weights, into saved buffers the next bwd uses
  bool keep_dgrad = false, dgrad_ready = false;
  void *wd1s = nullptr, *wd2s = nullptr, *wdscs = nullptr;
  void prep(hipStream_t st, const Params& P, void* sn_ws, bool for_bwd = false);
  // prep's work as job lists, for a network to launch all of its modules'
  // SN weights and packs together (pack_jobs with for_bwd marks the
  // data-gradient packs ready)
  void sn_jobs(const Params& P, std::vector<SnJob>& out);
  void pack_jobs(const Params& P, bool for_bwd, std::vector<PackJob>& out);
  void fwd(const Exec& ex, const Params& P, const void* x, const float* cond, void* y);
  // dcond_accumulate: add to dcond instead of overwriting it
  void bwd(const Exec& ex, const Params& P, const void* x, const float* cond, const void* dy, void* dx,
           float* dcond, bool dcond_accumulate);
};

// ----------------------------------------------------------- D block
struct DBlock {
  int B, H, W, cin, cout, npi;
  bool preact, down, lsc, f32;
  // the input is an image in 3x3-patch form (img_to_im2col, 9 cin <= 32
  // channels): conv1 runs as a 1x1 conv over the patches, the skip reads
  // the centre tap, and dx is the fp32 image gradient [B][H][W][4]
  bool im2col = false;
  float sn_eps;
  int Cip, Cop, Ho, Wo;
  SNSlot sn[3];
  void *wp1 = nullptr, *wp2 = nullptr, *wpsc = nullptr;
  void* h = nullptr;
  void* xp = nullptr;   // 2x2 average of the input (downsampling learnable skip)
  // conv2 + 2x2 average pool as one stride-2 4x4 conv (bf16 downsampling blocks)
  bool s2conv() const { return down && !f32; }
  // its data gradient as four sub-pixel 2x2 convs (K = 4 Cout) at every
  // width, so that forward and data gradient use the same bf16 folded taps
  // (the 3x3 form over the upsampled gradient would round the 3x3 taps)
  bool subdgrad() const { return s2conv(); }
  void plan_saved(Arena& a);
  size_t ws_size(int n_cu) const;
  // The forward's SN power iterations and weight packing: fwd runs them
  // itself unless prepped is set (then prep ran them before, e.g. on
  // another stream; sn_ws: sn_ws_all of the layout, or the block's share)
  bool prepped = false;
  bool keep_dgrad = false, dgrad_ready = false;   // as in GBlock
  void *wd1s = nullptr, *wd2s = nullptr, *wdscs = nullptr;
  void prep(hipStream_t st, const Params& P, void* sn_ws, bool for_bwd = false);
  void sn_jobs(const Params& P, std::vector<SnJob>& out);                       // as in GBlock
  void pack_jobs(const Params& P, bool for_bwd, std::vector<PackJob>& out);
  void fwd(const Exec& ex, const Params& P, const void* x, void* y);
  // dx may be null; dx_f32 writes an unrounded fp32 input gradient;
  // wgrad = false computes the input gradient only (no parameter gradients).
  void bwd(const Exec& ex, const Params& P, const void* x, const void* dy, void* dx, bool dx_f32,
           bool wgrad = true);
};

// ----------------------------------------------------------- attention
struct Attn {
  int B, H, W, C, npi;
  float sn_eps;
  int Cp, dk, dv, Nqkv;      // padded head dims; Nqkv = 2*dk + dv
  SNSlot sn[4];
  void *wqkv = nullptr, *wo = nullptr;   // packed fwd weights
  void *qkv = nullptr;       // [B][H][W][Nqkv] bf16 projections (pre-pool)
  void *kp = nullptr, *vp = nullptr;   // pooled keys / values
  void *o = nullptr;         // attention output [B][HW][dv] bf16
  float* o32 = nullptr;      // the same in fp32 for the backward's row term dO . O, in the
                             // attention kernels' register layout ([B][HWp / 32][dv / 32][4][64][4])
  float* lse = nullptr;      // [B][HWp] log2-sum-exp2 of the scores
  void plan_saved(Arena& a);
  size_t ws_size(int n_cu) const;
  // for_bwd = false: no backward will follow (o32 is not written)
  // The forward's SN power iterations and weight packing: fwd runs them
  // itself unless prepped is set (then prep ran them before, e.g. on
  // another stream; sn_ws: sn_ws_all of the layout, or the block's share)
  bool prepped = false;
  void prep(hipStream_t st, const Params& P, void* sn_ws);
  // as in GBlock; the attention packs divide by sigma, so they must follow
  // the SN launches of sn_jobs on the stream
  void sn_jobs(const Params& P, std::vector<SnJob>& out);
  void pack_jobs(const Params& P, std::vector<PackJob>& out);
  void fwd(const Exec& ex, const Params& P, const void* x, void* y, bool for_bwd = true);
  void bwd(const Exec& ex, const Params& P, const void* x, const void* dy, void* dx, bool wgrad = true);
};

// SN of one weight into a slot (power iteration updates u in place).
void sn_forward(const Exec& ex, const Params& P, const std::string& name, SNSlot& s, int npi, float eps);
// Group job descriptors: the power iteration of a named weight into a slot
// (persistent u in place, the slot keeps a copy), and its backward writing
// the weight's gradient from dwp (dL/d(W/sigma), padded layout, channel
// stride Cp) scaled by *scale (1 if null).
SnJob sn_job(const Params& P, const std::string& name, SNSlot& s);
SnBwdJob sn_bwd_job(const Params& P, const std::string& name, const SNSlot& s, const float* dwp, int R, int Cp,
                    const float* scale);
// workspace of a group of (rows, cols) weights
size_t sn_group_ws(const int64_t (*rc)[2], int n);
// workspace for any group of a layout's SN weights
size_t sn_ws_all(const Layout& L);

}  // namespace pg
