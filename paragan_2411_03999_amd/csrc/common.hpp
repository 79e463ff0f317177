// Shared device/host helpers for libparagan (gfx950 only).
#pragma once
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <string>

#define PG_DEV __device__ __forceinline__

namespace pg {

typedef uint16_t bf16_t;                                     // storage type
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));   // MFMA operand
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kCPad = 32;   // channel padding: the K depth of one bf16 MFMA step pair

__host__ __device__ inline int64_t cpad(int64_t c) { return (c + kCPad - 1) / kCPad * kCPad; }
__host__ __device__ inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// fp32 -> bf16, round to nearest even (NaN stays NaN): gfx950's
// v_cvt_pk_bf16_f32, two values per instruction.
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2v __attribute__((ext_vector_type(2)));
PG_DEV bf16_t f2bf(float f) { return __builtin_bit_cast(bf16_t, (__bf16)f); }
PG_DEV uint32_t f2bf2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){a, b}, bf16x2v));
}
PG_DEV float bf2f(bf16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

// 8 packed bf16 in a uint4 <-> 8 floats
PG_DEV void unpack8(const uint4& q, float* f) {
  const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = __uint_as_float(w[i] << 16);
    f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}
PG_DEV uint4 pack8(const float* f) {
  return make_uint4(f2bf2(f[0], f[1]), f2bf2(f[2], f[3]), f2bf2(f[4], f[5]), f2bf2(f[6], f[7]));
}

// Raw buffer loads (gfx9 buffer resource: base, byte size, raw 32-bit
// dwords).  A byte offset at or beyond the size reads zeros without touching
// memory, so out-of-range rows need no branch: they get kOOB.
constexpr uint32_t kOOB = 0xF0000000u;        // offsets from here on are out of range
constexpr int64_t kBufMax = 0xF0000000LL;      // largest buffer (bytes) addressable this way
PG_DEV __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int64_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)(uint32_t)bytes, 0x00020000);
}
PG_DEV uint4 buf_ld16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0));
}

// ReLU on 8 packed bf16 by their bit patterns: a negative bf16 is a negative
// int16, so max(v, 0) as packed int16 zeroes exactly the negatives (and -0).
typedef short short2v __attribute__((ext_vector_type(2)));
PG_DEV uint32_t relu2_bits(uint32_t w) {
  short2v v = __builtin_bit_cast(short2v, w);
  v = __builtin_elementwise_max(v, (short2v){0, 0});
  return __builtin_bit_cast(uint32_t, v);
}
PG_DEV uint4 relu8_bits(const uint4& q) {
  return make_uint4(relu2_bits(q.x), relu2_bits(q.y), relu2_bits(q.z), relu2_bits(q.w));
}

// element load/store for the two activation types
template <typename T> PG_DEV float ld(const T* p, int64_t i);
template <> PG_DEV float ld<float>(const float* p, int64_t i) { return p[i]; }
template <> PG_DEV float ld<bf16_t>(const bf16_t* p, int64_t i) { return bf2f(p[i]); }
template <typename T> PG_DEV void st(T* p, int64_t i, float v);
template <> PG_DEV void st<float>(float* p, int64_t i, float v) { p[i] = v; }
template <> PG_DEV void st<bf16_t>(bf16_t* p, int64_t i, float v) { p[i] = f2bf(v); }
// rounding to the storage precision of T (identity for fp32)
template <typename T> PG_DEV float rnd(float v);
template <> PG_DEV float rnd<float>(float v) { return v; }
template <> PG_DEV float rnd<bf16_t>(float v) { return bf2f(f2bf(v)); }

// wavefront reduction (64 lanes), result valid in every lane
PG_DEV float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
PG_DEV double wave_sum_d(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

}  // namespace pg

// ---------------------------------------------------------------- host side
#include <vector>

namespace pg {
// Opt-in launch profiler: an event pair around each instrumented launch on
// the context's stream, with the launch's algorithmic FLOPs.  Read (and
// reset) through paragan_profile_read once the stream is idle.
struct ProfRec {
  std::string name;
  double flops;
  hipEvent_t a, b;
  double bytes = 0.0;   // algorithmic HBM bytes (bandwidth-bound kernels)
};
struct Profiler {
  bool on = false;
  bool detail = false;   // tag each record with its GEMM shape
  std::vector<ProfRec> recs;
  std::vector<hipEvent_t> pool;
  hipEvent_t ev() {
    if (!pool.empty()) {
      hipEvent_t e = pool.back();
      pool.pop_back();
      return e;
    }
    hipEvent_t e;
    (void)hipEventCreate(&e);
    return e;
  }
};
// set by the C-ABI entry points for the duration of a call
extern thread_local Profiler* t_prof;

struct ProfScope {
  Profiler* p;
  hipStream_t st;
  hipEvent_t a = nullptr;
  ProfScope(hipStream_t s) : p(t_prof), st(s) {
    if (p && p->on) {
      a = p->ev();
      (void)hipEventRecord(a, st);
    }
  }
  void done(const std::string& name, double flops, double bytes = 0.0) {
    if (!a) return;
    hipEvent_t b = p->ev();
    (void)hipEventRecord(b, st);
    p->recs.push_back(ProfRec{name, flops, a, b, bytes});
    a = nullptr;
  }
  // a bandwidth-bound launch: its algorithmic bytes instead of FLOPs
  void done_bytes(const std::string& name, double bytes) { done(name, 0.0, bytes); }
  // as done(), with the launch's GEMM shape appended in detail mode
  void done(const std::string& name, double flops, int64_t m, int64_t n, int64_t k) {
    if (!a) return;
    if (!p->detail) return done(name, flops);
    done(name + "[" + std::to_string(m) + "," + std::to_string(n) + "," + std::to_string(k) + "]", flops);
  }
};
}  // namespace pg

struct paragan_ctx {
  hipStream_t stream = nullptr;
  // a second stream (default priority) for work that overlaps the caller's
  // stream inside one call, and events to order the two; created on first
  // use, released with the context
  hipStream_t side = nullptr;
  hipEvent_t ev[4] = {nullptr, nullptr, nullptr, nullptr};
  // a third stream (default priority) for the weight gradients of the block
  // backwards inside the step calls, beside their data gradients, and the
  // fork / join events that order it; created on first use
  hipStream_t wside = nullptr;
  hipEvent_t wev[2] = {nullptr, nullptr};
  bool overlap_wgrad = false;   // use wside (paragan_set_overlap_wgrad)
  int device = 0;
  int n_cu = 0;
  void* sn_scratch = nullptr;   // the device's address of the library's SN scratch array
  std::string err;
  pg::Profiler prof;
};

namespace pg {

struct Error {
  int code;
  std::string msg;
};

#define PG_HIP(call)                                                        \
  do {                                                                      \
    hipError_t e_ = (call);                                                 \
    if (e_ != hipSuccess)                                                   \
      throw ::pg::Error{-4, std::string(#call) + ": " + hipGetErrorString(e_)}; \
  } while (0)

#define PG_CHECK(cond, msg)                                                 \
  do {                                                                      \
    if (!(cond)) throw ::pg::Error{-1, std::string(msg)};                   \
  } while (0)

#define PG_LAUNCH_CHECK() PG_HIP(hipGetLastError())

}  // namespace pg
