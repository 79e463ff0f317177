// C ABI of libparagan (include/paragan.h): argument validation, buffer
// planning, and dispatch into the block executors.  Every entry point
// catches all exceptions and turns them into status codes.
#include <cstring>

#include "../../include/paragan.h"
#include "blocks.hpp"
#include "net.hpp"
#include <cmath>

using namespace pg;

static std::string g_create_err;

namespace {
// binds the context's profiler to the launchers for the duration of a call
struct ProfBind {
  explicit ProfBind(paragan_ctx* c) { pg::t_prof = c ? &c->prof : nullptr; }
  ~ProfBind() { pg::t_prof = nullptr; }
};
}  // namespace

static int fail(paragan_ctx* ctx, int code, const std::string& msg) {
  if (ctx) {
    ctx->err = msg;
    // leave no work of a failed call running on the context's own streams
    // (it may read the caller's buffers)
    if (ctx->side) (void)hipStreamSynchronize(ctx->side);
    if (ctx->wside) (void)hipStreamSynchronize(ctx->wside);
  } else {
    g_create_err = msg;
  }
  return code;
}

#define PG_TRY(ctx, ...)                                   \
  try {                                                    \
    __VA_ARGS__;                                           \
    return PARAGAN_OK;                                     \
  } catch (const ::pg::Error& e) {                         \
    return fail(ctx, e.code, e.msg);                       \
  } catch (const std::exception& e) {                      \
    return fail(ctx, PARAGAN_EINVAL, e.what());            \
  } catch (...) {                                          \
    return fail(ctx, PARAGAN_EINVAL, "unknown error");     \
  }

extern "C" {

int paragan_create(paragan_ctx** out, void* hip_stream) {
  if (!out) return fail(nullptr, PARAGAN_EINVAL, "paragan_create: out is NULL");
  try {
    int dev = 0;
    PG_HIP(hipGetDevice(&dev));
    hipDeviceProp_t p;
    PG_HIP(hipGetDeviceProperties(&p, dev));
    if (std::strncmp(p.gcnArchName, "gfx950", 6) != 0)
      throw Error{PARAGAN_EUNSUPPORTED, std::string("paragan needs gfx950, found ") + p.gcnArchName};
    void* scr = sn_scratch_init(dev);
    auto* c = new paragan_ctx;
    c->stream = (hipStream_t)hip_stream;
    c->device = dev;
    c->n_cu = p.multiProcessorCount;
    c->sn_scratch = scr;
    *out = c;
    return PARAGAN_OK;
  } catch (const Error& e) {
    return fail(nullptr, e.code, e.msg);
  }
}

void paragan_destroy(paragan_ctx* ctx) {
  if (!ctx) return;
  if (ctx->side) {
    (void)hipStreamSynchronize(ctx->side);
    (void)hipStreamDestroy(ctx->side);
  }
  if (ctx->wside) {
    (void)hipStreamSynchronize(ctx->wside);
    (void)hipStreamDestroy(ctx->wside);
  }
  for (hipEvent_t e : ctx->ev)
    if (e) (void)hipEventDestroy(e);
  for (hipEvent_t e : ctx->wev)
    if (e) (void)hipEventDestroy(e);
  delete ctx;
}

const char* paragan_last_error(const paragan_ctx* ctx) {
  return ctx ? ctx->err.c_str() : g_create_err.c_str();
}

int paragan_sync(paragan_ctx* ctx) {
  if (!ctx) return PARAGAN_EINVAL;
  PG_TRY(ctx, PG_HIP(hipStreamSynchronize(ctx->stream)))
}

int paragan_set_overlap_wgrad(paragan_ctx* ctx, int on) {
  if (!ctx) return PARAGAN_EINVAL;
  if (on != 0 && on != 1) return fail(ctx, PARAGAN_EINVAL, "paragan_set_overlap_wgrad: on must be 0 or 1");
  ctx->overlap_wgrad = on == 1;
  return PARAGAN_OK;
}

int64_t paragan_cpad(int64_t c) { return cpad(c); }

}  // extern "C"

// ------------------------------------------------------------ helpers
static void need(const void* p, const char* what) {
  if (!p) throw Error{PARAGAN_EINVAL, std::string(what) + " is NULL"};
}
static void aligned(const void* p, const char* what) {
  if (((uintptr_t)p & 255) != 0) throw Error{PARAGAN_EINVAL, std::string(what) + " is not 256-byte aligned"};
}

static int export_layout(const Layout& L, paragan_tensor_info* out, int32_t cap, int32_t* count,
                         int64_t* n_params, int64_t* n_u) {
  if (count) *count = (int32_t)L.e.size();
  if (n_params) *n_params = L.n_params;
  if (n_u) *n_u = L.n_u;
  if (out) {
    if (cap < (int32_t)L.e.size()) return PARAGAN_EINVAL;
    for (size_t i = 0; i < L.e.size(); ++i) {
      const Entry& e = L.e[i];
      paragan_tensor_info& t = out[i];
      std::memset(&t, 0, sizeof(t));
      std::strncpy(t.name, e.name.c_str(), sizeof(t.name) - 1);
      t.ndim = (int32_t)e.shape.size();
      for (size_t d = 0; d < e.shape.size() && d < 4; ++d) t.shape[d] = e.shape[d];
      t.offset = e.offset;
      t.u_offset = e.u_offset;
    }
  }
  return PARAGAN_OK;
}

// ------------------------------------------------------------ G block
static void gcheck(const paragan_gblock_desc* d) {
  if (!d) throw Error{PARAGAN_EINVAL, "gblock: desc is NULL"};
  PG_CHECK(d->B >= 1 && d->H >= 1 && d->W >= 1, "gblock: B, H, W must be >= 1");
  PG_CHECK(d->cin >= 1 && d->cout >= 1 && d->dc >= 1, "gblock: cin, cout, dc must be >= 1");
  PG_CHECK(d->dtype == PARAGAN_BF16 || d->dtype == PARAGAN_F32, "gblock: dtype must be PARAGAN_BF16 or PARAGAN_F32");
  PG_CHECK(d->n_power_iter >= 1, "gblock: n_power_iter must be >= 1");
  PG_CHECK(d->bn_eps > 0.f && d->sn_eps > 0.f, "gblock: eps must be > 0");
  PG_CHECK((int64_t)d->B * 4 * d->H * d->W < (1LL << 31), "gblock: too many output pixels");
}

static GBlock make_g(const paragan_gblock_desc* d) {
  GBlock g;
  g.B = d->B; g.H = d->H; g.W = d->W; g.cin = d->cin; g.cout = d->cout; g.dc = d->dc;
  g.npi = d->n_power_iter; g.f32 = d->dtype == PARAGAN_F32; g.bn_eps = d->bn_eps; g.sn_eps = d->sn_eps;
  Arena a(nullptr);
  g.plan_saved(a);
  return g;
}

extern "C" int paragan_gblock_check(const paragan_gblock_desc* d) { PG_TRY(nullptr, gcheck(d)) }

extern "C" int paragan_gblock_layout(const paragan_gblock_desc* d, paragan_tensor_info* out, int32_t cap,
                                     int32_t* count, int64_t* n_params, int64_t* n_u) {
  try {
    gcheck(d);
    return export_layout(gblock_layout(d->cin, d->cout, d->dc), out, cap, count, n_params, n_u);
  } catch (const Error& e) {
    return fail(nullptr, e.code, e.msg);
  }
}

extern "C" int paragan_gblock_sizes(const paragan_gblock_desc* d, size_t* saved, size_t* ws) {
  PG_TRY(nullptr, {
    gcheck(d);
    GBlock g = make_g(d);
    Arena a(nullptr);
    g.plan_saved(a);
    if (saved) *saved = a.off;
    int dev = 0, ncu = 256;
    if (hipGetDevice(&dev) == hipSuccess) {
      hipDeviceProp_t p;
      if (hipGetDeviceProperties(&p, dev) == hipSuccess) ncu = p.multiProcessorCount;
    }
    if (ws) *ws = g.ws_size(ncu);
  })
}

static size_t g_ws_for(paragan_ctx* ctx, const GBlock& g) { return g.ws_size(ctx->n_cu); }

extern "C" int paragan_gblock_fwd(paragan_ctx* ctx, const paragan_gblock_desc* d, const float* params, float* u,
                                  const void* x, const float* cond, void* y, void* saved, void* ws) {
  if (!ctx) return PARAGAN_EINVAL;
  ProfBind pb(ctx);
  PG_TRY(ctx, {
    gcheck(d);
    need(params, "params"); need(u, "u"); need(x, "x"); need(cond, "cond"); need(y, "y");
    need(saved, "saved"); need(ws, "ws");
    aligned(saved, "saved"); aligned(ws, "ws");
    GBlock g = make_g(d);
    Arena a(saved);
    g.plan_saved(a);
    Layout L = gblock_layout(d->cin, d->cout, d->dc);
    Params P{&L, "", params, u, nullptr};
    Exec ex{ctx->stream, ctx->n_cu, ws, g_ws_for(ctx, g)};
    g.fwd(ex, P, x, cond, y);
  })
}

extern "C" int paragan_gblock_bwd(paragan_ctx* ctx, const paragan_gblock_desc* d, const float* params,
                                  const void* x, const float* cond, const void* saved, const void* dy, void* dx,
                                  float* dcond, float* grads, void* ws) {
  if (!ctx) return PARAGAN_EINVAL;
  ProfBind pb(ctx);
  PG_TRY(ctx, {
    gcheck(d);
    need(params, "params"); need(x, "x"); need(cond, "cond"); need(saved, "saved"); need(dy, "dy");
    need(dx, "dx"); need(dcond, "dcond"); need(grads, "grads"); need(ws, "ws");
    aligned(saved, "saved"); aligned(ws, "ws");
    GBlock g = make_g(d);
    Arena a((void*)saved);
    g.plan_saved(a);
    Layout L = gblock_layout(d->cin, d->cout, d->dc);
    Params P{&L, "", params, nullptr, grads};
    Exec ex{ctx->stream, ctx->n_cu, ws, g_ws_for(ctx, g)};
    g.bwd(ex, P, x, cond, dy, dx, dcond, false);
  })
}

// ------------------------------------------------------------ D block
static void dcheck(const paragan_dblock_desc* d) {
  if (!d) throw Error{PARAGAN_EINVAL, "dblock: desc is NULL"};
  PG_CHECK(d->B >= 1 && d->H >= 1 && d->W >= 1, "dblock: B, H, W must be >= 1");
  PG_CHECK(d->cin >= 1 && d->cout >= 1, "dblock: cin, cout must be >= 1");
  PG_CHECK(d->dtype == PARAGAN_BF16 || d->dtype == PARAGAN_F32, "dblock: dtype must be PARAGAN_BF16 or PARAGAN_F32");
  PG_CHECK(d->n_power_iter >= 1, "dblock: n_power_iter must be >= 1");
  PG_CHECK(d->sn_eps > 0.f, "dblock: sn_eps must be > 0");
  PG_CHECK(!d->downsample || (d->H % 2 == 0 && d->W % 2 == 0), "dblock: pooling needs even H and W");
  PG_CHECK(d->learnable_sc || (d->cin == d->cout && !d->downsample),
           "dblock: an identity skip needs cin == cout and no pooling");
  PG_CHECK((int64_t)d->B * d->H * d->W < (1LL << 31), "dblock: too many pixels");
}

static DBlock make_d(const paragan_dblock_desc* d) {
  DBlock b;
  b.B = d->B; b.H = d->H; b.W = d->W; b.cin = d->cin; b.cout = d->cout; b.npi = d->n_power_iter;
  b.preact = d->preact != 0; b.down = d->downsample != 0; b.lsc = d->learnable_sc != 0;
  b.f32 = d->dtype == PARAGAN_F32; b.sn_eps = d->sn_eps;
  Arena a(nullptr);
  b.plan_saved(a);
  return b;
}

extern "C" int paragan_dblock_check(const paragan_dblock_desc* d) { PG_TRY(nullptr, dcheck(d)) }

extern "C" int paragan_dblock_layout(const paragan_dblock_desc* d, paragan_tensor_info* out, int32_t cap,
                                     int32_t* count, int64_t* n_params, int64_t* n_u) {
  try {
    dcheck(d);
    return export_layout(dblock_layout(d->cin, d->cout, d->learnable_sc != 0), out, cap, count, n_params, n_u);
  } catch (const Error& e) {
    return fail(nullptr, e.code, e.msg);
  }
}

static int device_cus() {
  int dev = 0, ncu = 256;
  if (hipGetDevice(&dev) == hipSuccess) {
    hipDeviceProp_t p;
    if (hipGetDeviceProperties(&p, dev) == hipSuccess) ncu = p.multiProcessorCount;
  }
  return ncu;
}

extern "C" int paragan_dblock_sizes(const paragan_dblock_desc* d, size_t* saved, size_t* ws) {
  PG_TRY(nullptr, {
    dcheck(d);
    DBlock b = make_d(d);
    Arena a(nullptr);
    b.plan_saved(a);
    if (saved) *saved = a.off;
    if (ws) *ws = b.ws_size(device_cus());
  })
}

extern "C" int paragan_dblock_fwd(paragan_ctx* ctx, const paragan_dblock_desc* d, const float* params, float* u,
                                  const void* x, void* y, void* saved, void* ws) {
  if (!ctx) return PARAGAN_EINVAL;
  ProfBind pb(ctx);
  PG_TRY(ctx, {
    dcheck(d);
    need(params, "params"); need(u, "u"); need(x, "x"); need(y, "y"); need(saved, "saved"); need(ws, "ws");
    aligned(saved, "saved"); aligned(ws, "ws");
    DBlock b = make_d(d);
    Arena a(saved);
    b.plan_saved(a);
    Layout L = dblock_layout(d->cin, d->cout, d->learnable_sc != 0);
    Params P{&L, "", params, u, nullptr};
    Exec ex{ctx->stream, ctx->n_cu, ws, b.ws_size(ctx->n_cu)};
    b.fwd(ex, P, x, y);
  })
}

extern "C" int paragan_dblock_bwd(paragan_ctx* ctx, const paragan_dblock_desc* d, const float* params,
                                  const void* x, const void* saved, const void* dy, void* dx, float* grads,
                                  void* ws) {
  if (!ctx) return PARAGAN_EINVAL;
  ProfBind pb(ctx);
  PG_TRY(ctx, {
    dcheck(d);
    need(params, "params"); need(x, "x"); need(saved, "saved"); need(dy, "dy"); need(grads, "grads");
    need(ws, "ws");
    aligned(saved, "saved"); aligned(ws, "ws");
    DBlock b = make_d(d);
    Arena a((void*)saved);
    b.plan_saved(a);
    Layout L = dblock_layout(d->cin, d->cout, d->learnable_sc != 0);
    Params P{&L, "", params, nullptr, grads};
    Exec ex{ctx->stream, ctx->n_cu, ws, b.ws_size(ctx->n_cu)};
    b.bwd(ex, P, x, dy, dx, false);
  })
}

// ------------------------------------------------------------ SN
extern "C" int paragan_sn_ws_size(int64_t rows, int64_t cols, size_t* ws_bytes) {
  PG_TRY(nullptr, {
    PG_CHECK(rows >= 1 && cols >= 1, "sn_ws_size: rows and cols must be >= 1");
    need(ws_bytes, "ws_bytes");
    *ws_bytes = sn_ws_bytes(rows, cols);
  })
}

static void sn_check(int64_t rows, int64_t cols, int n_iter, float eps) {
  PG_CHECK(rows >= 1 && cols >= 1, "sn_power_iter: rows and cols must be >= 1");
  PG_CHECK(n_iter >= 1, "sn_power_iter: n_iter must be >= 1");
  PG_CHECK(eps > 0.f, "sn_power_iter: eps must be > 0");
  PG_CHECK(rows < (1LL << 31) && cols < (1LL << 31), "sn_power_iter: matrix too large");
}

extern "C" int paragan_sn_check(int64_t rows, int64_t cols, int n_iter, float eps) {
  PG_TRY(nullptr, sn_check(rows, cols, n_iter, eps))
}

extern "C" int paragan_sn_power_iter(paragan_ctx* ctx, const float* W, int64_t rows, int64_t cols, float* u,
                                     float* v, float* sigma, int n_iter, float eps, void* ws) {
  if (!ctx) return PARAGAN_EINVAL;
  ProfBind pb(ctx);
  PG_TRY(ctx, {
    need(W, "W"); need(u, "u"); need(v, "v"); need(sigma, "sigma"); need(ws, "ws");
    aligned(ws, "ws");
    sn_check(rows, cols, n_iter, eps);
    sn_power_iter(ctx->stream, W, rows, cols, u, v, sigma, n_iter, eps, ws);
  })
}

extern "C" int paragan_sn_power_iter_noalloc(paragan_ctx* ctx, const float* W, int64_t rows, int64_t cols,
                                             float* u, float* v, float* sigma, int n_iter, float eps) {
  if (!ctx) return PARAGAN_EINVAL;
  PG_TRY(ctx, {
    need(W, "W"); need(u, "u"); need(v, "v"); need(sigma, "sigma");
    sn_check(rows, cols, n_iter, eps);
    const size_t want = sn_ws_bytes(rows, cols);
    PG_CHECK(want <= kSnScratchBytes, "sn_power_iter_noalloc: a " + std::to_string(rows) + " x " +
                                          std::to_string(cols) + " weight needs " + std::to_string(want) +
                                          " bytes of scratch, more than the library's " +
                                          std::to_string(kSnScratchBytes) + " (use paragan_sn_power_iter)");
    PG_CHECK(ctx->sn_scratch != nullptr, "sn_power_iter_noalloc: context has no scratch address");
    sn_power_iter(ctx->stream, W, rows, cols, u, v, sigma, n_iter, eps, ctx->sn_scratch);
  })
}

// ------------------------------------------------------------ attention
static void acheck(const paragan_attn_desc* d) {
  if (!d) throw Error{PARAGAN_EINVAL, "attn: desc is NULL"};
  PG_CHECK(d->B >= 1 && d->H >= 2 && d->W >= 2 && d->H % 2 == 0 && d->W % 2 == 0,
           "attn: B >= 1 and H, W even and >= 2");
  PG_CHECK(d->C >= 8 && d->C % 8 == 0, "attn: C must be a multiple of 8");
  PG_CHECK(d->C / 8 <= 32, "attn: C/8 query width above 32 is not supported");
  const int64_t dv = cpad(d->C / 2);
  PG_CHECK(dv == 32 || dv == 64 || dv == 96 || dv == 128, "attn: C/2 value width must pad to 32, 64, 96 or 128");
  PG_CHECK(d->n_power_iter >= 1 && d->sn_eps > 0.f, "attn: bad n_power_iter / sn_eps");
  PG_CHECK((int64_t)d->B * d->H * d->W < (1LL << 31), "attn: too many pixels");
}

static Attn make_a(const paragan_attn_desc* d) {
  Attn t;
  t.B = d->B; t.H = d->H; t.W = d->W; t.C = d->C; t.npi = d->n_power_iter; t.sn_eps = d->sn_eps;
  Arena a(nullptr);
  t.plan_saved(a);
  return t;
}

extern "C" int paragan_attn_check(const paragan_attn_desc* d) { PG_TRY(nullptr, acheck(d)) }

extern "C" int paragan_attn_layout(const paragan_attn_desc* d, paragan_tensor_info* out, int32_t cap,
                                   int32_t* count, int64_t* n_params, int64_t* n_u) {
  try {
    acheck(d);
    return export_layout(attn_layout(d->C), out, cap, count, n_params, n_u);
  } catch (const Error& e) {
    return fail(nullptr, e.code, e.msg);
  }
}

extern "C" int paragan_attn_sizes(const paragan_attn_desc* d, size_t* saved, size_t* ws) {
  PG_TRY(nullptr, {
    acheck(d);
    Attn t = make_a(d);
    Arena a(nullptr);
    t.plan_saved(a);
    if (saved) *saved = a.off;
    if (ws) *ws = t.ws_size(device_cus());
  })
}

extern "C" int paragan_attn_fwd(paragan_ctx* ctx, const paragan_attn_desc* d, const float* params, float* u,
                                const void* x, void* y, void* saved, void* ws) {
  if (!ctx) return PARAGAN_EINVAL;
  ProfBind pb(ctx);
  PG_TRY(ctx, {
    acheck(d);
    need(params, "params"); need(u, "u"); need(x, "x"); need(y, "y"); need(saved, "saved"); need(ws, "ws");
    aligned(saved, "saved"); aligned(ws, "ws");
    Attn t = make_a(d);
    Arena a(saved);
    t.plan_saved(a);
    Layout L = attn_layout(d->C);
    Params P{&L, "", params, u, nullptr};
    Exec ex{ctx->stream, ctx->n_cu, ws, t.ws_size(ctx->n_cu)};
    t.fwd(ex, P, x, y);
  })
}

extern "C" int paragan_attn_bwd(paragan_ctx* ctx, const paragan_attn_desc* d, const float* params, const void* x,
                                const void* saved, const void* dy, void* dx, float* grads, void* ws) {
  if (!ctx) return PARAGAN_EINVAL;
  ProfBind pb(ctx);
  PG_TRY(ctx, {
    acheck(d);
    need(params, "params"); need(x, "x"); need(saved, "saved"); need(dy, "dy"); need(dx, "dx");
    need(grads, "grads"); need(ws, "ws");
    aligned(saved, "saved"); aligned(ws, "ws");
    Attn t = make_a(d);
    Arena a((void*)saved);
    t.plan_saved(a);
    Layout L = attn_layout(d->C);
    Params P{&L, "", params, nullptr, grads};
    Exec ex{ctx->stream, ctx->n_cu, ws, t.ws_size(ctx->n_cu)};
    t.bwd(ex, P, x, dy, dx, true);
  })
}

// ------------------------------------------------------------ generator output layer
static void ocheck(const paragan_gout_desc* d) {
  if (!d) throw Error{PARAGAN_EINVAL, "gout: desc is NULL"};
  PG_CHECK(d->B >= 1 && d->H >= 1 && d->W >= 1 && d->C >= 1, "gout: B, H, W, C >= 1");
  PG_CHECK(ghead_shape_ok(d->W, d->C), "gout: needs cpad(C) <= 128, W a multiple of 4 and W small enough for the "
                                       "weight-gradient tile");
  PG_CHECK(d->n_power_iter >= 1 && d->bn_eps > 0.f && d->sn_eps > 0.f, "gout: bad n_power_iter / eps");
  PG_CHECK((int64_t)d->B * d->H * d->W < (1LL << 31), "gout: too many pixels");
}

static GOut make_o(const paragan_gout_desc* d) {
  GOut g;
  g.B = d->B; g.H = d->H; g.W = d->W; g.C = d->C; g.npi = d->n_power_iter;
  g.bn_eps = d->bn_eps; g.sn_eps = d->sn_eps;
  return g;
}

extern "C" int paragan_gout_check(const paragan_gout_desc* d) { PG_TRY(nullptr, ocheck(d)) }

extern "C" int paragan_gout_layout(const paragan_gout_desc* d, paragan_tensor_info* out, int32_t cap,
                                   int32_t* count, int64_t* n_params, int64_t* n_u) {
  try {
    ocheck(d);
    return export_layout(gout_layout(d->C), out, cap, count, n_params, n_u);
  } catch (const Error& e) {
    return fail(nullptr, e.code, e.msg);
  }
}

extern "C" int paragan_gout_sizes(const paragan_gout_desc* d, size_t* saved, size_t* ws) {
  PG_TRY(nullptr, {
    ocheck(d);
    GOut g = make_o(d);
    Arena a(nullptr);
    g.plan_saved(a);
    if (saved) *saved = a.off;
    if (ws) *ws = g.ws_size();
  })
}

extern "C" int paragan_gout_fwd(paragan_ctx* ctx, const paragan_gout_desc* d, const float* params, float* u,
                                const void* x, float* img, void* saved, void* ws) {
  if (!ctx) return PARAGAN_EINVAL;
  ProfBind pb(ctx);
  PG_TRY(ctx, {
    ocheck(d);
    need(params, "params"); need(u, "u"); need(x, "x"); need(img, "img"); need(saved, "saved"); need(ws, "ws");
    aligned(saved, "saved"); aligned(ws, "ws");
    GOut g = make_o(d);
    Arena a(saved);
    g.plan_saved(a);
    Layout L = gout_layout(d->C);
    Params P{&L, "", params, u, nullptr};
    g.fwd(Exec{ctx->stream, ctx->n_cu, ws, g.ws_size()}, P, x, img);
  })
}

extern "C" int paragan_gout_bwd(paragan_ctx* ctx, const paragan_gout_desc* d, const float* params, const void* x,
                                const float* img, const void* saved, const float* dimg, void* dx, float* grads,
                                void* ws) {
  if (!ctx) return PARAGAN_EINVAL;
  ProfBind pb(ctx);
  PG_TRY(ctx, {
    ocheck(d);
    need(params, "params"); need(x, "x"); need(img, "img"); need(saved, "saved"); need(dimg, "dimg");
    need(dx, "dx"); need(grads, "grads"); need(ws, "ws");
    aligned(saved, "saved"); aligned(ws, "ws");
    GOut g = make_o(d);
    Arena a((void*)saved);
    g.plan_saved(a);
    Layout L = gout_layout(d->C);
    Params P{&L, "", params, nullptr, grads};
    g.bwd(Exec{ctx->stream, ctx->n_cu, ws, g.ws_size()}, P, x, img, dimg, 3, dx);
  })
}

// ------------------------------------------------------------ networks, step
extern "C" int paragan_biggan_check(const paragan_biggan_desc* d) { PG_TRY(nullptr, check_arch(d)) }

extern "C" int paragan_net_layout(const paragan_biggan_desc* d, int32_t which, paragan_tensor_info* out,
                                  int32_t cap, int32_t* count, int64_t* n_params, int64_t* n_u) {
  try {
    check_arch(d);
    PG_CHECK(which == 0 || which == 1, "net_layout: which must be 0 (G) or 1 (D)");
    const Arch a = arch_from(d);
    return export_layout(which == 0 ? g_layout(a) : d_layout(a), out, cap, count, n_params, n_u);
  } catch (const Error& e) {
    return fail(nullptr, e.code, e.msg);
  }
}

extern "C" int paragan_train_step_ws_size(const paragan_biggan_desc* d, size_t* ws_bytes) {
  PG_TRY(nullptr, {
    check_arch(d);
    need(ws_bytes, "ws_bytes");
    *ws_bytes = train_step_ws(d, device_cus());
  })
}

static void need_state(const paragan_net_state* s, const char* who) {
  need(s, who);
  need(s->params, "params"); need(s->u, "u"); need(s->grads, "grads");
  need(s->opt_m, "opt_m"); need(s->opt_v, "opt_v");
  PG_CHECK(s->opt_t >= 0, "opt_t must be >= 0");
}

static int finish_losses(paragan_ctx* ctx, const float* losses, int n, const char* who) {
  for (int k = 0; k < n; ++k)
    if (!std::isfinite(losses[k])) return fail(ctx, PARAGAN_ENONFINITE, std::string(who) + ": non-finite loss");
  return PARAGAN_OK;
}

#define PG_STEP_TRY(ctx, ...)                              \
  try {                                                    \
    __VA_ARGS__;                                           \
  } catch (const ::pg::Error& e) {                         \
    return fail(ctx, e.code, e.msg);                       \
  } catch (const std::exception& e) {                      \
    return fail(ctx, PARAGAN_EINVAL, e.what());            \
  }

extern "C" int paragan_g_sample(paragan_ctx* ctx, const paragan_biggan_desc* d, paragan_net_state* G,
                                const float* z, const int32_t* y, float* img, void* ws) {
  if (!ctx) return PARAGAN_EINVAL;
  ProfBind pb(ctx);
  PG_TRY(ctx, {
    check_arch(d);
    need_state(G, "G");
    need(z, "z"); need(y, "y"); need(img, "img"); need(ws, "ws");
    aligned(ws, "ws");
    g_sample(ctx, d, G, z, y, img, ws);
  })
}

extern "C" int paragan_d_step(paragan_ctx* ctx, const paragan_biggan_desc* d, paragan_net_state* D,
                              const float* x_real, const int32_t* y_real, const float* x_fake,
                              const int32_t* y_fake, void* ws, float* loss_host) {
  if (!ctx) return PARAGAN_EINVAL;
  ProfBind pb(ctx);
  PG_STEP_TRY(ctx, {
    check_arch(d);
    need_state(D, "D");
    need(x_real, "x_real"); need(y_real, "y_real"); need(x_fake, "x_fake"); need(y_fake, "y_fake");
    need(ws, "ws"); need(loss_host, "loss_host");
    aligned(ws, "ws");
    d_step(ctx, d, D, x_real, y_real, x_fake, y_fake, ws, loss_host);
  })
  return finish_losses(ctx, loss_host, 1, "d_step");
}

extern "C" int paragan_g_step(paragan_ctx* ctx, const paragan_biggan_desc* d, paragan_net_state* G,
                              paragan_net_state* D, const float* z, const int32_t* y, void* ws, float* loss_host) {
  if (!ctx) return PARAGAN_EINVAL;
  ProfBind pb(ctx);
  PG_STEP_TRY(ctx, {
    check_arch(d);
    need_state(G, "G");
    need_state(D, "D");
    need(z, "z"); need(y, "y"); need(ws, "ws"); need(loss_host, "loss_host");
    aligned(ws, "ws");
    g_step(ctx, d, G, D, z, y, ws, loss_host);
  })
  return finish_losses(ctx, loss_host, 1, "g_step");
}

extern "C" int paragan_train_step(paragan_ctx* ctx, const paragan_biggan_desc* d, paragan_net_state* G,
                                  paragan_net_state* D, const paragan_step_inputs* in, int32_t n_D, void* ws,
                                  float* losses_host) {
  if (!ctx) return PARAGAN_EINVAL;
  ProfBind pb(ctx);
  PG_STEP_TRY(ctx, {
    check_arch(d);
    need_state(G, "G");
    need_state(D, "D");
    need(in, "inputs"); need(ws, "ws"); need(losses_host, "losses_host");
    aligned(ws, "ws");
    PG_CHECK(n_D >= 1 && n_D <= 63, "train_step: n_D must be in [1, 63]");
    need(in->x_real, "x_real"); need(in->y_real, "y_real"); need(in->z_fake, "z_fake"); need(in->y_fake, "y_fake");
    for (int k = 0; k < n_D; ++k) {
      need(in->x_real[k], "x_real[k]"); need(in->y_real[k], "y_real[k]");
      need(in->z_fake[k], "z_fake[k]"); need(in->y_fake[k], "y_fake[k]");
    }
    need(in->z_g, "z_g"); need(in->y_g, "y_g");
    train_step(ctx, d, G, D, in, n_D, ws, losses_host);
  })
  return finish_losses(ctx, losses_host, n_D + 1, "train_step");
}

extern "C" int paragan_async_ws_size(const paragan_biggan_desc* d, int32_t n_D, size_t* ws_bytes) {
  PG_TRY(nullptr, {
    check_arch(d);
    need(ws_bytes, "ws_bytes");
    PG_CHECK(n_D >= 1 && n_D <= 63, "async_ws_size: n_D must be in [1, 63]");
    *ws_bytes = async_step_ws(d, n_D, device_cus());
  })
}

extern "C" int paragan_async_step(paragan_ctx* ctx, const paragan_biggan_desc* d, paragan_net_state* G,
                                  paragan_net_state* D, const paragan_async_inputs* in, int32_t n_D, void* ws,
                                  float* losses_host) {
  if (!ctx) return PARAGAN_EINVAL;
  ProfBind pb(ctx);
  PG_STEP_TRY(ctx, {
    check_arch(d);
    need_state(G, "G");
    need_state(D, "D");
    need(in, "inputs"); need(ws, "ws"); need(losses_host, "losses_host");
    aligned(ws, "ws");
    PG_CHECK(n_D >= 1 && n_D <= 63, "async_step: n_D must be in [1, 63]");
    PG_CHECK((int64_t)n_D * d->B * d->img * d->img < (1LL << 31), "async_step: generator batch n_D * B too large");
    need(in->x_real, "x_real"); need(in->y_real, "y_real");
    for (int k = 0; k < n_D; ++k) { need(in->x_real[k], "x_real[k]"); need(in->y_real[k], "y_real[k]"); }
    need(in->z, "z"); need(in->y, "y");
    need(in->img_buff, "img_buff"); need(in->lab_buff, "lab_buff"); need(in->pred_buff, "pred_buff");
    async_step(ctx, d, G, D, in, n_D, ws, losses_host);
  })
  return finish_losses(ctx, losses_host, n_D + 1, "async_step");
}

// ------------------------------------------------------------ profiler
extern "C" int paragan_profile(paragan_ctx* ctx, int enable) {
  if (!ctx) return PARAGAN_EINVAL;
  ctx->prof.on = enable != 0;
  ctx->prof.detail = enable == 2;
  return PARAGAN_OK;
}

extern "C" int paragan_profile_read(paragan_ctx* ctx, paragan_kernel_stat* out, int32_t cap, int32_t* count) {
  if (!ctx) return PARAGAN_EINVAL;
  PG_TRY(ctx, {
    need(count, "count");
    PG_HIP(hipStreamSynchronize(ctx->stream));
    std::vector<paragan_kernel_stat> agg;
    for (auto& r : ctx->prof.recs) {
      float ms = 0.f;
      PG_HIP(hipEventElapsedTime(&ms, r.a, r.b));
      paragan_kernel_stat* k = nullptr;
      for (auto& x : agg)
        if (r.name == x.name) k = &x;
      if (!k) {
        agg.push_back(paragan_kernel_stat{});
        k = &agg.back();
        std::strncpy(k->name, r.name.c_str(), sizeof(k->name) - 1);
      }
      k->launches += 1;
      k->total_ms += ms;
      k->flops += r.flops;
      k->bytes += r.bytes;
      ctx->prof.pool.push_back(r.a);
      ctx->prof.pool.push_back(r.b);
    }
    ctx->prof.recs.clear();
    *count = (int32_t)agg.size();
    if (out)
      for (int32_t i = 0; i < *count && i < cap; ++i) out[i] = agg[i];
  })
}
