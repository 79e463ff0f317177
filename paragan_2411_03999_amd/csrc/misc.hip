// Bandwidth-bound kernels: spectral normalisation (power iteration, weight
// packing, backward), batch-norm statistics / affine tables / backward,
// bias-gradient column sums.  All reductions run in a fixed order (no float
// atomics), so results are bitwise reproducible run to run.
#include "misc.hpp"

#include <mutex>

namespace pg {

// ----------------------------------------------------- block reductions
template <int NT>
PG_DEV float block_sum(float v, float* sh) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) sh[w] = v;
  __syncthreads();
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < NT / 64; ++i) s += sh[i];
  __syncthreads();
  return s;
}
template <int NT>
PG_DEV double block_sum_d(double v, double* sh) {
  v = wave_sum_d(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) sh[w] = v;
  __syncthreads();
  double s = 0.0;
#pragma unroll
  for (int i = 0; i < NT / 64; ++i) s += sh[i];
  __syncthreads();
  return s;
}

// ------------------------------------------------ spectral normalisation
// The power iteration of every SN weight of a module runs as one group:
// one launch per phase for all of its weights (a module has up to
// kSnGroupMax), each launch finding its weight from a block-offset table
// passed by value with the job descriptors.
//   phase 1  part[j][c] = sum_{r in row chunk j} W[r][c] u[r]
//   phase 2  t[c] = sum_j part[j][c] (fixed order), and per-block partials of |t|^2
//   phase 3  s'[r] = W[r] . t                                              (a wave per row)
//   phase 4  (a block per weight) v = t / max(|t|, eps), s = s' / max(|t|, eps),
//            u = s / max(|s|, eps), sigma = u . s
// (W v = (W t) / max(|t|, eps) exactly; only the rounding order differs from
// normalising t first.)  Phase 1 tiles W as (row chunk) x (cw columns): a
// block's threads are P = 256 / cw row lanes of cw columns, so a matrix with
// few columns (a linear map from a 20-d z chunk) still reads whole rows per
// step; the P lane sums combine in order through LDS.  Row chunks are many
// for narrow matrices (about 1024 blocks in all), so phase 2 splits each
// column's chunk sum over L = 256 / cw2 lanes, combined in lane order (cw2
// = 64 columns per block when there are more than 32 chunks, else 256).
struct SnJobK {
  const float* W;
  float *u, *v, *sigma, *u_save, *part, *s;
  double* tsq;          // per-block partials of |t|^2 (ceil(cols / cw2))
  int rows, cols, rchunk, nrc, cw, P, cw2;
};
struct SnGroupK {
  SnJobK j[kSnGroupMax];
  int n;
  int off[kSnGroupMax + 1];   // first block of each job in this launch
};

PG_DEV int find_job(const int* off, int n, int bid) {
  int i = 0;
  while (i + 1 < n && bid >= off[i + 1]) ++i;
  return i;
}

__global__ __launch_bounds__(256) void k_sng_wtu(SnGroupK g) {
  __shared__ float sh[256];
  const int i = find_job(g.off, g.n, blockIdx.x);
  const SnJobK& J = g.j[i];
  const int lb = blockIdx.x - g.off[i];
  const int cb = (J.cols + J.cw - 1) / J.cw;
  const int rc = lb / cb;
  const int cc = (int)threadIdx.x % J.cw, ro = (int)threadIdx.x / J.cw;
  const int c = (lb - rc * cb) * J.cw + cc;
  const bool on = ro < J.P && c < J.cols;
  const int r0 = rc * J.rchunk, r1 = min(r0 + J.rchunk, J.rows);
  float acc = 0.f;
  if (on) {
    const int64_t ld = J.cols, st = (int64_t)J.P * ld;
    const float* W = J.W + (int64_t)(r0 + ro) * ld + c;
    // four independent chains: four rows in flight per thread
    float s0 = 0.f, s1 = 0.f, s2 = 0.f, s3 = 0.f;
    int r = r0 + ro;
    for (; r + 3 * J.P < r1; r += 4 * J.P, W += 4 * st) {
      s0 = fmaf(W[0], J.u[r], s0);
      s1 = fmaf(W[st], J.u[r + J.P], s1);
      s2 = fmaf(W[2 * st], J.u[r + 2 * J.P], s2);
      s3 = fmaf(W[3 * st], J.u[r + 3 * J.P], s3);
    }
    for (; r < r1; r += J.P, W += st) s0 = fmaf(W[0], J.u[r], s0);
    acc = (s0 + s1) + (s2 + s3);
  }
  if (J.P == 1) {
    if (on) J.part[(int64_t)rc * J.cols + c] = acc;
    return;
  }
  sh[threadIdx.x] = acc;
  __syncthreads();
  if (ro == 0 && c < J.cols) {
    float t = 0.f;
    for (int k = 0; k < J.P; ++k) t += sh[k * J.cw + cc];
    J.part[(int64_t)rc * J.cols + c] = t;
  }
}

__global__ __launch_bounds__(256) void k_sng_t(SnGroupK g) {
  __shared__ float sh[256];
  __shared__ double shd[4];
  const int i = find_job(g.off, g.n, blockIdx.x);
  const SnJobK& J = g.j[i];
  const int lb = blockIdx.x - g.off[i];
  const int cw2 = J.cw2, L = 256 / cw2;
  const int cc = (int)threadIdx.x % cw2, ln = (int)threadIdx.x / cw2;
  const int c = lb * cw2 + cc;
  float t = 0.f;
  if (ln < L && c < J.cols)
    for (int j = ln; j < J.nrc; j += L) t += J.part[(int64_t)j * J.cols + c];
  sh[threadIdx.x] = t;
  __syncthreads();
  float tc = 0.f;
  if (ln == 0 && c < J.cols) {
    for (int k = 0; k < L; ++k) tc += sh[k * cw2 + cc];
    J.v[c] = tc;
  }
  const double ss = block_sum_d<256>((double)tc * tc, shd);
  if (threadIdx.x == 0) J.tsq[lb] = ss;
}

__global__ __launch_bounds__(256) void k_sng_wv(SnGroupK g) {
  const int i = find_job(g.off, g.n, blockIdx.x);
  const SnJobK& J = g.j[i];
  const int r = (blockIdx.x - g.off[i]) * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (r >= J.rows) return;
  const float* W = J.W + (int64_t)r * J.cols;
  float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
  int c = lane;
  for (; c + 192 < J.cols; c += 256) {
    a0 = fmaf(W[c], J.v[c], a0);
    a1 = fmaf(W[c + 64], J.v[c + 64], a1);
    a2 = fmaf(W[c + 128], J.v[c + 128], a2);
    a3 = fmaf(W[c + 192], J.v[c + 192], a3);
  }
  for (; c < J.cols; c += 64) a0 = fmaf(W[c], J.v[c], a0);
  const float acc = wave_sum((a0 + a1) + (a2 + a3));
  if (lane == 0) J.s[r] = acc;
}

__global__ __launch_bounds__(1024) void k_sng_u(SnGroupK g, float eps) {
  __shared__ double sh[16];
  __shared__ float inv_t_sh;
  const SnJobK& J = g.j[blockIdx.x];
  {
    const int nb = (J.cols + J.cw2 - 1) / J.cw2;
    double tt = 0.0;
    for (int b = threadIdx.x; b < nb; b += 1024) tt += J.tsq[b];
    tt = block_sum_d<1024>(tt, sh);
    if (threadIdx.x == 0) inv_t_sh = 1.f / fmaxf((float)sqrt(tt), eps);
  }
  __syncthreads();
  const float inv_t = inv_t_sh;
  for (int c = threadIdx.x; c < J.cols; c += 1024) J.v[c] = J.v[c] * inv_t;
  double ss = 0.0;
  for (int r = threadIdx.x; r < J.rows; r += 1024) {
    const float sr = J.s[r] * inv_t;
    ss += (double)sr * sr;
  }
  const double tot = block_sum_d<1024>(ss, sh);
  const float inv = 1.f / fmaxf((float)sqrt(tot), eps);
  double sg = 0.0;
  for (int r = threadIdx.x; r < J.rows; r += 1024) {
    const float sr = J.s[r] * inv_t;
    const float un = sr * inv;
    J.u[r] = un;
    if (J.u_save) J.u_save[r] = un;
    sg += (double)un * sr;
  }
  const double sgt = block_sum_d<1024>(sg, sh);
  if (threadIdx.x == 0) *J.sigma = (float)sgt;
}

// phase-1 tiling: cw columns x P row lanes per block, nrc row chunks of rchunk rows
struct SnTiling {
  int cw, P, rchunk, nrc, cw2;
};
static SnTiling sn_tiling(int64_t rows, int64_t cols) {
  SnTiling t;
  t.cw = (int)std::min<int64_t>(cols, 256);
  t.P = 256 / t.cw;
  const int64_t cb = cdiv(cols, (int64_t)t.cw);
  // at least 8 rows per lane; about 1024 blocks over the column tiles
  const int64_t want = std::max<int64_t>(16, 1024 / cb);
  t.nrc = (int)std::max<int64_t>(1, std::min<int64_t>({want, 256, cdiv(rows, (int64_t)t.P * 8)}));
  t.rchunk = (int)cdiv(rows, (int64_t)t.nrc);
  t.nrc = (int)cdiv(rows, (int64_t)t.rchunk);
  t.cw2 = (int)std::min<int64_t>(cols, t.nrc > 32 ? 64 : 256);
  return t;
}

static size_t sn_job_ws(int64_t rows, int64_t cols) {
  const SnTiling t = sn_tiling(rows, cols);
  return align256((size_t)t.nrc * cols * 4) + align256((size_t)rows * 4) + align256((size_t)cdiv(cols, (int64_t)t.cw2) * 8);
}

size_t sn_ws_bytes(int64_t rows, int64_t cols) { return sn_job_ws(rows, cols); }

size_t sn_group_ws_bytes(const SnJob* jobs, int n) {
  size_t t = 0;
  for (int i = 0; i < n; ++i) t += sn_job_ws(jobs[i].rows, jobs[i].cols);
  return t;
}

void sn_power_iter_group(hipStream_t st, const SnJob* jobs, int n, int n_iter, float eps, void* ws) {
  PG_CHECK(n >= 1 && n <= kSnGroupMax, "sn group: 1.." + std::to_string(kSnGroupMax) + " weights");
  SnGroupK g{};
  g.n = n;
  char* w = (char*)ws;
  for (int i = 0; i < n; ++i) {
    const SnJob& a = jobs[i];
    PG_CHECK(a.rows >= 1 && a.cols >= 1 && a.rows < (1LL << 31) && a.cols < (1LL << 31), "sn group: shape");
    SnJobK& k = g.j[i];
    k.W = a.W; k.u = a.u; k.v = a.v; k.sigma = a.sigma; k.u_save = nullptr;
    k.rows = (int)a.rows; k.cols = (int)a.cols;
    const SnTiling tl = sn_tiling(a.rows, a.cols);
    k.cw = tl.cw; k.P = tl.P; k.rchunk = tl.rchunk; k.nrc = tl.nrc; k.cw2 = tl.cw2;
    k.part = (float*)w;
    k.s = (float*)(w + align256((size_t)k.nrc * a.cols * 4));
    k.tsq = (double*)(w + align256((size_t)k.nrc * a.cols * 4) + align256((size_t)a.rows * 4));
    w += sn_job_ws(a.rows, a.cols);
  }
  int b1 = 0, b2 = 0, b3 = 0;
  int o1[kSnGroupMax + 1], o2[kSnGroupMax + 1], o3[kSnGroupMax + 1];
  for (int i = 0; i < n; ++i) {
    o1[i] = b1;
    o2[i] = b2;
    o3[i] = b3;
    b1 += (int)cdiv(g.j[i].cols, g.j[i].cw) * g.j[i].nrc;
    b2 += (int)cdiv(g.j[i].cols, g.j[i].cw2);
    b3 += (int)cdiv(g.j[i].rows, 4);
  }
  o1[n] = b1;
  o2[n] = b2;
  o3[n] = b3;
  // algorithmic bytes: each matvec streams W once (plus its vectors); the
  // normalisations move only vectors
  double wbytes = 0.0, vbytes = 0.0;
  for (int i = 0; i < n; ++i) {
    wbytes += 4.0 * ((double)jobs[i].rows * jobs[i].cols + jobs[i].rows + jobs[i].cols);
    vbytes += 4.0 * (2.0 * jobs[i].rows + 2.0 * jobs[i].cols);
  }
  for (int it = 0; it < n_iter; ++it) {
    if (it + 1 == n_iter)
      for (int i = 0; i < n; ++i) g.j[i].u_save = jobs[i].u_save;
    std::copy(o1, o1 + n + 1, g.off);
    {
      ProfScope ps(st);
      hipLaunchKernelGGL(k_sng_wtu, dim3(b1), dim3(256), 0, st, g);
      ps.done_bytes("k_sng_wtu", wbytes);
    }
    std::copy(o2, o2 + n + 1, g.off);
    {
      ProfScope ps(st);
      hipLaunchKernelGGL(k_sng_t, dim3(b2), dim3(256), 0, st, g);
      ps.done_bytes("k_sng_t", vbytes);
    }
    std::copy(o3, o3 + n + 1, g.off);
    {
      ProfScope ps(st);
      hipLaunchKernelGGL(k_sng_wv, dim3(b3), dim3(256), 0, st, g);
      ps.done_bytes("k_sng_wv", wbytes);
    }
    {
      ProfScope ps(st);
      hipLaunchKernelGGL(k_sng_u, dim3(n), dim3(1024), 0, st, g, eps);
      ps.done_bytes("k_sng_u", vbytes);
    }
  }
  PG_LAUNCH_CHECK();
}

// Scratch of the allocation-free SN entry point.  In host code `scratch`
// names a host-side stand-in, not the array: its device address comes from
// hipGetSymbolAddress, once per device (each device holds its own copy), and
// only that address is ever handed to a kernel.  The kernels write every
// byte of the scratch they read, so it needs no clearing between calls.
static __device__ __align__(256) unsigned char scratch[kSnScratchBytes];
constexpr int kScratchDevices = 64;
static std::mutex g_scratch_mu;
static void* g_scratch_ptr[kScratchDevices] = {};

void* sn_scratch_init(int device) {
  PG_CHECK(device >= 0 && device < kScratchDevices, "sn scratch: device ordinal out of range");
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[device]) {
    void* p = nullptr;
    PG_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    PG_CHECK(p != nullptr && ((uintptr_t)p & 255) == 0, "sn scratch: symbol address not 256-byte aligned");
    g_scratch_ptr[device] = p;
  }
  return g_scratch_ptr[device];
}

void sn_power_iter_all(hipStream_t st, const SnJob* jobs, int n, int n_iter, float eps, void* ws) {
  for (int i = 0; i < n; i += kSnGroupMax) {
    const int k = std::min(kSnGroupMax, n - i);
    sn_power_iter_group(st, jobs + i, k, n_iter, eps, ws);
    ws = (char*)ws + sn_group_ws_bytes(jobs + i, k);
  }
}

void sn_power_iter(hipStream_t st, const float* W, int64_t rows, int64_t cols, float* u, float* v,
                   float* sigma, int n_iter, float eps, void* ws, float* u_save) {
  const SnJob j{W, rows, cols, u, v, sigma, u_save};
  sn_power_iter_group(st, &j, 1, n_iter, eps, ws);
}

// Pack W/sigma into the conv operand layouts, every weight of a group in
// one launch.
//  forward: dst[n][r][s][c]  ([Np][R][R][Cp]),  n < Cout, c < Cin (else 0)
//  dgrad:   dst[c][r][s][n]  ([Cp][R][R][Np]) = W[n][R-1-r][R-1-s][c]
//  pool4:   dst[n][u][v][c]  ([Np][4][4][Cp]) = 1/4 sum over a, b in {0, 1}
//           of W[n][u-a][v-b][c] (terms inside the 3x3 filter only)
//  dsum4:   dst[c][u][v][n]  ([Cp][4][4][Np]) = sum over a, b in {0, 1}
//           of W[n][2-u+a][2-v+b][c] (terms inside the filter only)
//  sub:     dst[p][n][du][dv][c] ([4][Np][2][2][Cp]), p = 2a + b, = sum of
//           W[n][r][s][c] over r in S(a, du), s in S(b, dv), where S(a, 0) =
//           [0, a] and S(a, 1) = [1 + a, 2]
//  subdg:   dst[p][c][du][dv][n] ([4][Cp][2][2][Np]) = the same sums of
//           W[n][2-r][2-s][c]
//  rep4:    dst[c][u][v][n]  ([Cp][2][2][Np]) = W[n][c] (a 1x1 filter)
// The forward layout is a padded copy (a thread per element, both sides
// contiguous along c); the dgrad layout transposes (n, c) per tap through
// a 32 x 32 LDS tile so that reads run along c and writes along n.
struct PackJobK {
  const float* W;
  const float* sigma;
  void* dst;
  int Cout, Cin, R, Np, Cp, mode;
  int wvec;   // filter rows are whole float4s (Cin % 4 == 0, koff % 4 == 0)
  int koff;   // destination channel of input channel 0 (fwd and dgrad modes)
};
struct PackGroupK {
  PackJobK j[kSnGroupMax];
  int n;
  int off[kSnGroupMax + 1];
};

template <typename T>
PG_DEV void store8f(T* p, const float* v);
template <>
PG_DEV void store8f<bf16_t>(bf16_t* p, const float* v) {
  *reinterpret_cast<uint4*>(p) = pack8(v);
}
template <>
PG_DEV void store8f<float>(float* p, const float* v) {
  *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
  *reinterpret_cast<float4*>(p + 4) = make_float4(v[4], v[5], v[6], v[7]);
}

template <typename T>
PG_DEV void store4f(T* p, const float* v);
template <>
PG_DEV void store4f<bf16_t>(bf16_t* p, const float* v) {
  *reinterpret_cast<uint2*>(p) = make_uint2(f2bf2(v[0], v[1]), f2bf2(v[2], v[3]));
}
template <>
PG_DEV void store4f<float>(float* p, const float* v) {
  *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
}

// four consecutive channels c .. c + 3 of filter row `row` (zeros past Cin):
// one 16-byte load when the rows are whole float4s.  A tensor of the flat
// parameter buffer starts at any float offset; global memory accepts the
// unaligned vector access.
PG_DEV void ld4w(const float* W, int64_t row, int Cin, int c, bool wvec, float* v) {
  const float* p = W + row * Cin + c;
  if (wvec && c + 4 <= Cin) {
    const float4 f = *reinterpret_cast<const float4*>(p);
    v[0] = f.x; v[1] = f.y; v[2] = f.z; v[3] = f.w;
  } else {
#pragma unroll
    for (int q = 0; q < 4; ++q) v[q] = c + q < Cin ? p[q] : 0.f;
  }
}

// A folded tap (a sum of up to four fp32 filter taps, times an optional
// 1/sigma and 1/4) rounded once to the stored type: the sum is formed in
// double, where it is exact, and rounded from there, so the stored value is
// the correctly rounded folded tap.  bf16: round to nearest even at bit 45
// of the double pattern (8 significant bits kept; a carry into the exponent
// is the next power of two); below bf16's normal range (no filter tap of
// these models) through fp32.
template <typename T>
PG_DEV float round_fold(double v);
template <>
PG_DEV float round_fold<float>(double v) {
  return (float)v;
}
template <>
PG_DEV float round_fold<bf16_t>(double v) {
  unsigned long long b = (unsigned long long)__double_as_longlong(v);
  const unsigned e = (unsigned)((b >> 52) & 0x7ff);
  if (e == 0x7ff || e < 1023 - 126) return bf2f(f2bf((float)v));
  b += ((1ull << 44) - 1) + ((b >> 45) & 1ull);
  b &= ~((1ull << 45) - 1);
  return (float)__longlong_as_double((long long)b);
}

template <typename T>
__global__ __launch_bounds__(256) void k_pack_group(PackGroupK g) {
  __shared__ float tile[64][65];
  const int i = find_job(g.off, g.n, blockIdx.x);
  const PackJobK& J = g.j[i];
  const int lb = blockIdx.x - g.off[i];
  const int RR = J.R * J.R;
  // a null sigma packs the filter unnormalised (the convolution then
  // divides its accumulator by sigma)
  const float inv = J.sigma ? 1.f / *J.sigma : 1.f;
  T* dst = (T*)J.dst;
  if (J.mode == kPackPool4) {
    // four consecutive channels of one (n, u, v) per thread
    const int e = (lb * 256 + (int)threadIdx.x) * 4;
    if (e >= J.Np * 16 * J.Cp) return;
    const int t = e / J.Cp;     // n * 16 + u * 4 + v
    const int c = e - t * J.Cp;
    const int n = t >> 4, u = (t >> 2) & 3, v = t & 3;
    double acc[4] = {0.0, 0.0, 0.0, 0.0};
    if (n < J.Cout && c < J.Cin) {
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b2 = 0; b2 < 2; ++b2) {
          const int r = u - a, s_ = v - b2;
          if (r >= 0 && r < 3 && s_ >= 0 && s_ < 3) {
            float w4[4];
            ld4w(J.W, (int64_t)n * 9 + r * 3 + s_, J.Cin, c, J.wvec, w4);
#pragma unroll
            for (int q = 0; q < 4; ++q) acc[q] += (double)w4[q];
          }
        }
    }
    float out[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) out[q] = round_fold<T>(acc[q] * 0.25 * (double)inv);
    store4f<T>(dst + e, out);
    return;
  }
  if (J.mode == kPackSub) {
    // four consecutive channels of one (p, n, du, dv) per thread
    const int e = (lb * 256 + (int)threadIdx.x) * 4;
    if (e >= 4 * J.Np * 4 * J.Cp) return;
    const int t = e / J.Cp;   // (p * Np + n) * 4 + du * 2 + dv
    const int c = e - t * J.Cp;
    const int dv = t & 1, du = (t >> 1) & 1, pn = t >> 2;
    const int p = pn / J.Np, n = pn - p * J.Np;
    const int a = p >> 1, b2 = p & 1;
    const int r0 = du ? 1 + a : 0, r1 = du ? 2 : a, s0 = dv ? 1 + b2 : 0, s1 = dv ? 2 : b2;
    double acc[4] = {0.0, 0.0, 0.0, 0.0};
    if (n < J.Cout && c < J.Cin)
      for (int r = r0; r <= r1; ++r)
        for (int s_ = s0; s_ <= s1; ++s_) {
          float w4[4];
          ld4w(J.W, (int64_t)n * 9 + r * 3 + s_, J.Cin, c, J.wvec, w4);
#pragma unroll
          for (int q = 0; q < 4; ++q) acc[q] += (double)w4[q];
        }
    float out[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) out[q] = round_fold<T>(acc[q] * (double)inv);
    store4f<T>(dst + e, out);
    return;
  }
  if (J.mode == kPackFwd) {
    // 32-bit indices (the host checks the sizes): eight consecutive channels per thread
    const int e = (lb * 256 + (int)threadIdx.x) * 8;
    if (e >= J.Np * RR * J.Cp) return;
    const int t = e / J.Cp;     // n * RR + tap
    const int c = e - t * J.Cp;
    const int n = t / RR;
    const float* src = J.W + (int64_t)t * J.Cin;
    const int cs = c - J.koff;   // source channel of destination channel c
    float v[8];
    if (n < J.Cout && J.wvec && cs >= 0 && cs + 8 <= J.Cin) {
      const float4 a = *reinterpret_cast<const float4*>(src + cs), b = *reinterpret_cast<const float4*>(src + cs + 4);
      v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
    } else {
#pragma unroll
      for (int q = 0; q < 8; ++q) v[q] = (n < J.Cout && cs + q >= 0 && cs + q < J.Cin) ? src[cs + q] : 0.f;
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) v[q] *= inv;
    store8f<T>(dst + e, v);
    return;
  }
  // transposing modes: (n, c) tiles of 64 x 64 per destination tap through
  // LDS; a thread reads four consecutive c of four rows n and writes four
  // consecutive n of four rows c
  const int tn = (J.Np + 63) >> 6, tc = (J.Cp + 63) >> 6;
  const int tap = lb / (tn * tc);
  const int rem = lb - tap * tn * tc;
  const int n0 = (rem / tc) * 64, c0 = (rem % tc) * 64;
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  const int DR = J.mode == kPackDgradSum4 ? 4 : (J.mode == kPackSubDgrad || J.mode == kPackDgradRep4 ? 2 : J.R);
  const int DRR = DR * DR;
  const int p = tap / DRR, ptap = tap - p * DRR;   // parity class (sub-pixel mode), tap within it
  const int u = ptap / DR, v = ptap - u * DR;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int n = n0 + ty + 16 * k, cb = c0 + 4 * tx;
    double val[4] = {0.0, 0.0, 0.0, 0.0};
    if (n < J.Cout) {
      if (J.mode == kPackDgradSum4) {
        if (cb < J.Cin)
#pragma unroll
          for (int a = 0; a < 2; ++a)
#pragma unroll
            for (int b2 = 0; b2 < 2; ++b2) {
              const int r = 2 - u + a, s_ = 2 - v + b2;
              if (r >= 0 && r < 3 && s_ >= 0 && s_ < 3) {
                float w4[4];
                ld4w(J.W, (int64_t)n * 9 + r * 3 + s_, J.Cin, cb, J.wvec, w4);
#pragma unroll
                for (int q = 0; q < 4; ++q) val[q] += (double)w4[q];
              }
            }
      } else if (J.mode == kPackSubDgrad) {
        const int a = p >> 1, b2 = p & 1;
        const int r0 = u ? 1 + a : 0, r1 = u ? 2 : a, s0 = v ? 1 + b2 : 0, s1 = v ? 2 : b2;
        if (cb < J.Cin)
          for (int r = r0; r <= r1; ++r)
            for (int s_ = s0; s_ <= s1; ++s_) {
              float w4[4];
              ld4w(J.W, (int64_t)n * 9 + (2 - r) * 3 + (2 - s_), J.Cin, cb, J.wvec, w4);
#pragma unroll
              for (int q = 0; q < 4; ++q) val[q] += (double)w4[q];
            }
      } else {
        const int ftap = J.mode == kPackDgradRep4 ? 0 : (J.R - 1 - u) * J.R + (J.R - 1 - v);
        const int cs = cb - J.koff;   // source channel of destination channel cb
        const float* src = J.W + ((int64_t)n * RR + ftap) * J.Cin + cs;
        if (J.wvec && cs >= 0 && cs + 4 <= J.Cin) {
          const float4 f = *reinterpret_cast<const float4*>(src);
          val[0] = f.x; val[1] = f.y; val[2] = f.z; val[3] = f.w;
        } else {
#pragma unroll
          for (int q = 0; q < 4; ++q) val[q] = cs + q >= 0 && cs + q < J.Cin ? src[q] : 0.f;
        }
      }
    }
    // a single tap is an fp32 value already (times an fp32 1/sigma); a sum
    // of taps is rounded once from its exact double value
    const bool folded = J.mode == kPackDgradSum4 || J.mode == kPackSubDgrad;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      tile[ty + 16 * k][4 * tx + q] = folded ? round_fold<T>(val[q] * (double)inv) : (float)val[q] * inv;
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int c = c0 + ty + 16 * k, nb = n0 + 4 * tx;
    if (c < J.Cp && nb < J.Np) {
      const float w4[4] = {tile[4 * tx][ty + 16 * k], tile[4 * tx + 1][ty + 16 * k], tile[4 * tx + 2][ty + 16 * k],
                           tile[4 * tx + 3][ty + 16 * k]};
      store4f<T>(dst + (((int64_t)p * J.Cp + c) * DRR + ptap) * J.Np + nb, w4);
    }
  }
}

void pack_all(hipStream_t st, bool f32, const PackJob* jobs, int n) {
  for (int i = 0; i < n; i += kSnGroupMax) pack_group(st, f32, jobs + i, std::min(kSnGroupMax, n - i));
}

void pack_group(hipStream_t st, bool f32, const PackJob* jobs, int n) {
  PG_CHECK(n >= 1 && n <= kSnGroupMax, "pack group: 1.." + std::to_string(kSnGroupMax) + " weights");
  PackGroupK g{};
  g.n = n;
  int64_t b = 0;
  for (int i = 0; i < n; ++i) {
    const PackJob& a = jobs[i];
    PG_CHECK(a.koff == 0 || ((a.mode == kPackFwd || a.mode == kPackDgrad) && a.koff > 0 && a.koff + a.Cin <= a.Cp),
             "pack group: channel offset (fwd and dgrad modes, within Cp)");
    g.j[i] = PackJobK{a.W, a.sigma, a.dst, a.Cout, a.Cin, a.R, a.Np, a.Cp, a.mode,
                      a.Cin % 4 == 0 && a.koff % 4 == 0 ? 1 : 0, a.koff};
    g.off[i] = (int)b;
    const int RR = a.R * a.R;
    const bool four = a.mode == kPackPool4 || a.mode == kPackDgradSum4;
    const bool sub = a.mode == kPackSub || a.mode == kPackSubDgrad;
    const bool rep = a.mode == kPackDgradRep4;
    const int RRd = four || sub ? 16 : (rep ? 4 : RR);   // taps of the packed filter (all parities)
    PG_CHECK(!(four || sub) || a.R == 3, "pack group: the 4x4 and sub-pixel modes pack a 3x3 filter");
    PG_CHECK(!rep || a.R == 1, "pack group: the 2x2 replication packs a 1x1 filter");
    PG_CHECK(a.Cp % 4 == 0 && (int64_t)a.Np * RRd * a.Cp < (1LL << 31) &&
             (int64_t)a.Cout * RR * a.Cin < (1LL << 31), "pack group: shape");
    const bool tr = a.mode == kPackDgrad || a.mode == kPackDgradSum4 || a.mode == kPackSubDgrad || rep;
    PG_CHECK(!tr || a.Np % 4 == 0, "pack group: transposed rows of 4");
    PG_CHECK(tr || a.Cp % 8 == 0, "pack group: rows of 8");
    b += tr ? (int64_t)RRd * cdiv(a.Np, 64) * cdiv(a.Cp, 64)
            : (a.mode == kPackFwd ? cdiv((int64_t)a.Np * RRd * a.Cp, 2048) : cdiv((int64_t)a.Np * RRd * a.Cp, 1024));
    PG_CHECK(b < (1LL << 31), "pack group: too large");
  }
  g.off[n] = (int)b;
  // algorithmic bytes: the fp32 master weights read, the packed operand written
  double bytes = 0.0;
  for (int i = 0; i < n; ++i) {
    const PackJob& a = jobs[i];
    const bool four = a.mode == kPackPool4 || a.mode == kPackDgradSum4;
    const bool sub = a.mode == kPackSub || a.mode == kPackSubDgrad;
    const int RRd = four || sub ? 16 : (a.mode == kPackDgradRep4 ? 4 : a.R * a.R);
    bytes += 4.0 * a.Cout * a.R * a.R * a.Cin + (f32 ? 4.0 : 2.0) * a.Np * RRd * a.Cp;
  }
  ProfScope ps(st);
  if (f32)
    hipLaunchKernelGGL(k_pack_group<float>, dim3((unsigned)b), dim3(256), 0, st, g);
  else
    hipLaunchKernelGGL(k_pack_group<bf16_t>, dim3((unsigned)b), dim3(256), 0, st, g);
  ps.done_bytes("k_pack_group", bytes);
  PG_LAUNCH_CHECK();
}

void pack_weight(hipStream_t st, bool f32, const float* W, const float* sigma, int Cout, int Cin,
                 int R, int Np, int Cp, bool dgrad, void* dst) {
  const PackJob j{W, sigma, dst, Cout, Cin, R, Np, Cp, dgrad ? kPackDgrad : kPackFwd};
  pack_group(st, f32, &j, 1);
}

// Transposed 1x1 pack into columns [col_off, col_off + Np) of a [Cp][ld]
// matrix: dst[c][col_off + n] = W[n][c] / sigma (zero outside Cout x Cin).
template <typename T>
__global__ void k_pack_t(const float* W, const float* sigma, int Cout, int Cin, int Cp, int Np, int ld,
                         int col_off, T* dst) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (int64_t)Cp * Np) return;
  const int n = (int)(i % Np), c = (int)(i / Np);
  const float v = (n < Cout && c < Cin) ? W[(int64_t)n * Cin + c] / *sigma : 0.f;
  st<T>(dst, (int64_t)c * ld + col_off + n, v);
}

void pack_weight_t(hipStream_t st, bool f32, const float* W, const float* sigma, int Cout, int Cin, int Cp,
                   int Np, int ld, int col_off, void* dst) {
  dim3 g((unsigned)cdiv((int64_t)Cp * Np, 256));
  if (f32)
    hipLaunchKernelGGL(k_pack_t<float>, g, dim3(256), 0, st, W, sigma, Cout, Cin, Cp, Np, ld, col_off,
                       (float*)dst);
  else
    hipLaunchKernelGGL(k_pack_t<bf16_t>, g, dim3(256), 0, st, W, sigma, Cout, Cin, Cp, Np, ld, col_off,
                       (bf16_t*)dst);
  PG_LAUNCH_CHECK();
}

// Weight gradient of a 3x3 filter from that of its pooled stride-2 4x4 form
// (W4 = W * box / 4): dw[n][r][s][c] = 1/4 sum over a, b in {0, 1} of
// dw4[n][r+a][s+b][c]; both fp32 in the padded [Np][taps][Cp] layouts.
__global__ void k_fold_pool4(const float* dw4, int Np, int Cp, float* dw) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (int64_t)Np * 9 * Cp) return;
  const int c = (int)(i % Cp);
  const int64_t t = i / Cp;
  const int tap = (int)(t % 9), n = (int)(t / 9);
  const int r = tap / 3, s_ = tap % 3;
  const float* src = dw4 + (int64_t)n * 16 * Cp + c;
  const float v = (src[(r * 4 + s_) * Cp] + src[(r * 4 + s_ + 1) * Cp]) +
                  (src[((r + 1) * 4 + s_) * Cp] + src[((r + 1) * 4 + s_ + 1) * Cp]);
  dw[i] = 0.25f * v;
}

void fold_pool4_wgrad(hipStream_t st, const float* dw4, int Np, int Cp, float* dw) {
  hipLaunchKernelGGL(k_fold_pool4, dim3((unsigned)cdiv((int64_t)Np * 9 * Cp, 256)), dim3(256), 0, st, dw4, Np, Cp,
                     dw);
  PG_LAUNCH_CHECK();
}

// SN backward, every weight of a group in two launches.  dwp: dL/d(W/sigma)
// in the padded forward layout [Np][R][R][Cp]; W: master [Cout][R][R][Cin].
//   dW = (s dWsn - s <dWsn, W/sigma> u v^T) / sigma,  s = *scale (1 if null),
// v indexed by (r, s, c).  Launch 1 forms fixed-order block partials of
// <dWsn, W> (up to kSnbParts blocks per weight); launch 2 sums a weight's
// partials (the same order in every block) and applies the update.  Both
// take 4 consecutive elements of a row (tap) per thread when Cin % 4 == 0
// (16-byte accesses, one division per 4 elements), else one.
struct SnBwdJobK {
  const float *dwp, *W, *u, *v, *sigma, *scale;
  float *dW, *part;
  int Cout, Cin, RR, Cp, nparts, vec;
};
struct SnBwdGroupK {
  SnBwdJobK j[kSnGroupMax];
  int n;
  int off[kSnGroupMax + 1];
};

__global__ __launch_bounds__(256) void k_sngb_dot(SnBwdGroupK g) {
  __shared__ float sh[4];
  const int i = find_job(g.off, g.n, blockIdx.x);
  const SnBwdJobK& J = g.j[i];
  const int lb = blockIdx.x - g.off[i];
  const int total = J.Cout * J.RR * J.Cin;      // < 2^31 (host-checked)
  float acc = 0.f;
  if (J.vec) {
    const int q = total >> 2;                   // groups of 4 (Cin % 4 == 0)
    float a1 = 0.f;
    int e4 = lb * 256 + (int)threadIdx.x;
    const int step = J.nparts * 256;
    for (; e4 < q; e4 += step) {
      const int e = 4 * e4, t = e / J.Cin, c = e - t * J.Cin;
      const float4 d = *reinterpret_cast<const float4*>(J.dwp + (int64_t)t * J.Cp + c);
      const float4 w = *reinterpret_cast<const float4*>(J.W + e);
      acc = fmaf(d.x, w.x, acc);
      a1 = fmaf(d.y, w.y, a1);
      acc = fmaf(d.z, w.z, acc);
      a1 = fmaf(d.w, w.w, a1);
    }
    acc += a1;
  } else {
    for (int e = lb * 256 + (int)threadIdx.x; e < total; e += J.nparts * 256) {
      const int t = e / J.Cin;
      const int c = e - t * J.Cin;
      acc = fmaf(J.dwp[(int64_t)t * J.Cp + c], J.W[e], acc);
    }
  }
  const float s = block_sum<256>(acc, sh);
  if (threadIdx.x == 0) J.part[lb] = s;
}

__global__ __launch_bounds__(256) void k_sngb_apply(SnBwdGroupK g) {
  __shared__ float sh[4];
  const int i = find_job(g.off, g.n, blockIdx.x);
  const SnBwdJobK& J = g.j[i];
  const int lb = blockIdx.x - g.off[i];
  float p = 0.f;
  for (int k = (int)threadIdx.x; k < J.nparts; k += 256) p += J.part[k];
  const float sig = *J.sigma;
  const float extra = J.scale ? *J.scale : 1.f;
  const float dot = block_sum<256>(p, sh) / sig * extra;   // s <dWsn, W/sigma>
  const float inv = 1.f / sig;
  const int total = J.Cout * J.RR * J.Cin;
  const int per = J.vec ? 4 : 1;
  const int units = total / per;
  const int nb = g.off[i + 1] - g.off[i];
  for (int q = lb * 256 + (int)threadIdx.x; q < units; q += nb * 256) {
    const int e = q * per;
    const int t = e / J.Cin;        // n * RR + tap
    const int c = e - t * J.Cin;
    const int n = t / J.RR;
    const int k = e - n * J.RR * J.Cin;   // column index (tap, c)
    const float un = dot * J.u[n];
    if (J.vec) {
      const float4 d = *reinterpret_cast<const float4*>(J.dwp + (int64_t)t * J.Cp + c);
      const float4 v = *reinterpret_cast<const float4*>(J.v + k);
      *reinterpret_cast<float4*>(J.dW + e) = make_float4((extra * d.x - un * v.x) * inv, (extra * d.y - un * v.y) * inv,
                                                         (extra * d.z - un * v.z) * inv, (extra * d.w - un * v.w) * inv);
    } else {
      J.dW[e] = (extra * J.dwp[(int64_t)t * J.Cp + c] - un * J.v[k]) * inv;
    }
  }
}

void sn_bwd_group(hipStream_t st, const SnBwdJob* jobs, int n, float* part) {
  PG_CHECK(n >= 1 && n <= kSnGroupMax, "sn bwd group: 1.." + std::to_string(kSnGroupMax) + " weights");
  SnBwdGroupK g{};
  g.n = n;
  SnBwdGroupK g2;
  int b1 = 0;
  int64_t b2 = 0;
  for (int i = 0; i < n; ++i) {
    const SnBwdJob& a = jobs[i];
    const int64_t total = (int64_t)a.Cout * a.R * a.R * a.Cin;
    PG_CHECK(total < (1LL << 31) && (int64_t)a.Cout * a.R * a.R * a.Cp < (1LL << 40), "sn bwd group: shape");
    // 4-wide when rows are whole float4s in both layouts and the workspace
    // operands (dwp, v) are 16-byte aligned; W and dW sit in the flat
    // parameter buffers at any float offset (unaligned vector accesses)
    const bool vec = a.Cin % 4 == 0 && a.Cp % 4 == 0 && (((uintptr_t)a.dwp | (uintptr_t)a.v) & 15) == 0;
    const int64_t units = vec ? total / 4 : total;
    const int np = (int)std::max<int64_t>(1, std::min<int64_t>(kSnbParts, cdiv(units, 256 * 8)));
    g.j[i] = SnBwdJobK{a.dwp, a.W, a.u, a.v, a.sigma, a.scale, a.dW, part + (int64_t)i * kSnbParts,
                       a.Cout, a.Cin, a.R * a.R, a.Cp, np, vec ? 1 : 0};
    g.off[i] = b1;
    b1 += np;
  }
  g.off[n] = b1;
  g2 = g;
  for (int i = 0; i < n; ++i) {
    g2.off[i] = (int)b2;
    const int64_t total = (int64_t)g.j[i].Cout * g.j[i].RR * g.j[i].Cin;
    b2 += cdiv(g.j[i].vec ? total / 4 : total, 256 * 8);   // up to 8 units per thread
  }
  g2.off[n] = (int)b2;
  PG_CHECK(b2 < (1LL << 31), "sn bwd group: too large");
  // algorithmic bytes: <dW, W> reads both; the projection reads the raw
  // gradient and writes the parameter gradient
  double bytes = 0.0;
  for (int i = 0; i < n; ++i) bytes += 8.0 * jobs[i].Cout * jobs[i].R * jobs[i].R * jobs[i].Cin;
  {
    ProfScope ps(st);
    hipLaunchKernelGGL(k_sngb_dot, dim3(b1), dim3(256), 0, st, g);
    ps.done_bytes("k_sngb_dot", bytes);
  }
  {
    ProfScope ps(st);
    hipLaunchKernelGGL(k_sngb_apply, dim3((unsigned)b2), dim3(256), 0, st, g2);
    ps.done_bytes("k_sngb_apply", bytes);
  }
  PG_LAUNCH_CHECK();
}

void sn_bwd(hipStream_t st, const float* dwp, const float* W, const float* u, const float* v,
            const float* sigma, int Cout, int Cin, int R, int Cp, const float* scale, float* dW,
            float* part /* kSnbParts floats */) {
  const SnBwdJob j{dwp, W, u, v, sigma, scale, dW, Cout, Cin, R, Cp};
  sn_bwd_group(st, &j, 1, part);
}

// ------------------------------------------------ per-channel reductions
// Column sums and batch-norm statistics over the rows (pixels) of an NHWC
// tensor, in two fixed-order levels (bitwise reproducible, no atomics).
// Level 1: a block takes a chunk of rows; a thread owns 8 consecutive
// channels (one 16-byte bf16 load or two fp32 loads per row) of the rows
// ro, ro + P, ... of the chunk, P threads sharing each channel group.  The
// P partials per channel then combine in order through LDS.  Level 2 merges
// the chunks.  Chunks are sized so that there are at most kMaxChunks of
// them: enough blocks to fill the chip, few partials for level 2.  Statistics use shifted sums per thread (shift = the thread's
// first value, so the sums stay well conditioned) and Chan's parallel
// variance formula for every merge.
constexpr int kRowsPerThread = 32;   // minimum rows per thread
constexpr int kMaxChunks = 1024;

struct RedShape {
  int CC, P, rows_blk;
};
// C: channels reduced (real count); the reduction covers cpad(C) channels of M rows
inline RedShape red_shape(int C, int64_t M) {
  RedShape r;
  r.CC = (int)(cpad(C) / 8);
  r.P = std::max(1, 256 / r.CC);
  const int64_t rpt = std::max<int64_t>(kRowsPerThread, cdiv(M, (int64_t)kMaxChunks * r.P));
  r.rows_blk = (int)(r.P * rpt);
  return r;
}

template <typename T>
PG_DEV void load8f(const T* p, float* v);
template <>
PG_DEV void load8f<bf16_t>(const bf16_t* p, float* v) {
  unpack8(*reinterpret_cast<const uint4*>(p), v);
}
template <>
PG_DEV void load8f<float>(const float* p, float* v) {
  const float4 a = *reinterpret_cast<const float4*>(p), b = *reinterpret_cast<const float4*>(p + 4);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}

PG_DEV void chan_merge(double& n, double& mu, double& m2, double nb, double mb, double m2b) {
  if (nb <= 0.0) return;
  const double nn = n + nb;
  const double d = mb - mu;
  mu += d * nb / nn;
  m2 += m2b + d * d * n * nb / nn;
  n = nn;
}

// STATS: pa = chunk mean, pb = chunk M2; else pa = chunk sum.  [chunk][C]
template <typename T, bool STATS>
__global__ __launch_bounds__(256) void k_colred(const T* x, int64_t M, int C, int ldc, RedShape sh, float* pa,
                                                float* pb) {
  __shared__ float s_a[256 * 8], s_b[256 * 8];
  __shared__ int s_n[256];
  const int t = threadIdx.x;
  const int cc = t % sh.CC, ro = t / sh.CC;
  const int64_t r0 = (int64_t)blockIdx.x * sh.rows_blk;
  const int64_t r1 = r0 + sh.rows_blk < M ? r0 + sh.rows_blk : M;
  float sft[8], s1[8], s2[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) sft[e] = s1[e] = s2[e] = 0.f;
  int n = 0;
  if (ro < sh.P) {
    int64_t r = r0 + ro;
    if (STATS && r < r1) load8f<T>(x + r * ldc + cc * 8, sft);
    auto add = [&](const float* v) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float d = v[e] - sft[e];
        s1[e] += d;
        if (STATS) s2[e] = fmaf(d, d, s2[e]);
      }
      ++n;
    };
    // four rows in flight per thread, accumulated in row order
    for (; r + 3 * sh.P < r1; r += 4 * sh.P) {
      float v[4][8];
#pragma unroll
      for (int u = 0; u < 4; ++u) load8f<T>(x + (r + u * sh.P) * ldc + cc * 8, v[u]);
#pragma unroll
      for (int u = 0; u < 4; ++u) add(v[u]);
    }
    for (; r < r1; r += sh.P) {
      float v[8];
      load8f<T>(x + r * ldc + cc * 8, v);
      add(v);
    }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    if (STATS) {
      const float mu = n ? sft[e] + s1[e] / (float)n : 0.f;
      s_a[t * 8 + e] = mu;
      s_b[t * 8 + e] = n ? s2[e] - s1[e] * (s1[e] / (float)n) : 0.f;
    } else {
      s_a[t * 8 + e] = s1[e];
    }
  }
  s_n[t] = n;
  __syncthreads();
  for (int c = t; c < C; c += 256) {
    const int g = c >> 3, e = c & 7;
    if (STATS) {
      double nn = 0.0, mu = 0.0, m2 = 0.0;
      for (int j = 0; j < sh.P; ++j) {
        const int u = j * sh.CC + g;
        chan_merge(nn, mu, m2, (double)s_n[u], (double)s_a[u * 8 + e], (double)s_b[u * 8 + e]);
      }
      pa[(int64_t)blockIdx.x * C + c] = (float)mu;
      pb[(int64_t)blockIdx.x * C + c] = (float)m2;
    } else {
      float sum = 0.f;
      for (int j = 0; j < sh.P; ++j) sum += s_a[(j * sh.CC + g) * 8 + e];
      pa[(int64_t)blockIdx.x * C + c] = sum;
    }
  }
}

// fixed-order sum of the chunk partials: 16 channels per block, 64 lane
// groups summing every 64th chunk, then the 64 group sums in order
__global__ __launch_bounds__(1024) void k_colsum_fin(const float* part, int nch, int C, float scale, float* out) {
  __shared__ float sp[64][16];
  const int cl = threadIdx.x & 15, grp = threadIdx.x >> 4;
  const int c = blockIdx.x * 16 + cl;
  float s = 0.f;
  if (c < C)
    for (int j = grp; j < nch; j += 64) s += part[(int64_t)j * C + c];
  sp[grp][cl] = s;
  __syncthreads();
  if (grp == 0 && c < C) {
    float t = 0.f;
    for (int i = 0; i < 64; ++i) t += sp[i][cl];
    out[c] = t * scale;
  }
}

size_t colsum_ws_bytes(int64_t M, int C) {
  return align256((size_t)cdiv(M, red_shape(C, M).rows_blk) * C * 4);
}

void colsum(hipStream_t st, bool f32, const void* x, int64_t M, int C, int ldc, float scale, float* out,
            void* ws) {
  if (M <= 0) {
    fill(st, out, C, 0.f);
    return;
  }
  const RedShape sh = red_shape(C, M);
  PG_CHECK(ldc >= cpad(C) && ldc % 8 == 0, "colsum: channel stride");
  const int nch = (int)cdiv(M, sh.rows_blk);
  float* part = (float*)ws;
  ProfScope ps(st);
  if (f32)
    hipLaunchKernelGGL((k_colred<float, false>), dim3(nch), dim3(256), 0, st, (const float*)x, M, C, ldc, sh, part,
                       nullptr);
  else
    hipLaunchKernelGGL((k_colred<bf16_t, false>), dim3(nch), dim3(256), 0, st, (const bf16_t*)x, M, C, ldc, sh,
                       part, nullptr);
  hipLaunchKernelGGL(k_colsum_fin, dim3((unsigned)cdiv(C, 16)), dim3(1024), 0, st, part, nch, C, scale, out);
  ps.done_bytes("colsum", (double)M * C * (f32 ? 4 : 2));
  PG_LAUNCH_CHECK();
}

// ------------------------------------------------------- batch norm
// Merge of the chunk statistics, per channel c: with n_j rows, mean m_j and
// M2_j per chunk, mean = sum n_j m_j / M and M2 = sum (M2_j + n_j (m_j -
// mean)^2) -- two passes in fp64, no division per chunk.  A block takes 16
// channels; its 64 lane groups (lane / 16 + 4 wave) sum every 64th chunk,
// and the 64 group sums combine in group order.
__global__ __launch_bounds__(1024) void k_bn_fin(const float* pmean, const float* pm2, int nch, int rows_blk,
                                                 int64_t M, int C, float eps, float* mean, float* rstd) {
  __shared__ double sp[64][16];
  __shared__ double smu[16];
  const int cl = threadIdx.x & 15, grp = threadIdx.x >> 4;
  const int c = blockIdx.x * 16 + cl;
  const bool on = c < C;
  auto nrows = [&](int j) { return (double)std::min<int64_t>(rows_blk, M - (int64_t)j * rows_blk); };
  double s = 0.0;
  if (on)
    for (int j = grp; j < nch; j += 64) s += nrows(j) * (double)pmean[(int64_t)j * C + c];
  sp[grp][cl] = s;
  __syncthreads();
  if (grp == 0) {
    double t = 0.0;
    for (int i = 0; i < 64; ++i) t += sp[i][cl];
    smu[cl] = t / (double)M;
  }
  __syncthreads();
  const double mu = smu[cl];
  double q = 0.0;
  if (on)
    for (int j = grp; j < nch; j += 64) {
      const double d = (double)pmean[(int64_t)j * C + c] - mu;
      q += (double)pm2[(int64_t)j * C + c] + nrows(j) * d * d;
    }
  __syncthreads();
  sp[grp][cl] = q;
  __syncthreads();
  if (grp == 0 && on) {
    double t = 0.0;
    for (int i = 0; i < 64; ++i) t += sp[i][cl];
    mean[c] = (float)mu;
    rstd[c] = (float)(1.0 / sqrt(t / (double)M + (double)eps));
  }
}

size_t bn_stats_ws_bytes(int64_t M, int C) {
  return 2 * align256((size_t)cdiv(M, red_shape(C, M).rows_blk) * C * 4);
}

void bn_stats(hipStream_t st, bool f32, const void* x, int64_t M, int C, int ldc, float eps, float* mean,
              float* rstd, void* ws) {
  PG_CHECK(M > 0, "bn_stats: empty batch");
  const RedShape sh = red_shape(C, M);
  PG_CHECK(ldc >= cpad(C) && ldc % 8 == 0, "bn_stats: channel stride");
  const int nch = (int)cdiv(M, sh.rows_blk);
  float* pmean = (float*)ws;
  float* pm2 = (float*)((char*)ws + align256((size_t)nch * C * 4));
  ProfScope ps(st);
  if (f32)
    hipLaunchKernelGGL((k_colred<float, true>), dim3(nch), dim3(256), 0, st, (const float*)x, M, C, ldc, sh, pmean,
                       pm2);
  else
    hipLaunchKernelGGL((k_colred<bf16_t, true>), dim3(nch), dim3(256), 0, st, (const bf16_t*)x, M, C, ldc, sh,
                       pmean, pm2);
  hipLaunchKernelGGL(k_bn_fin, dim3((unsigned)cdiv(C, 16)), dim3(1024), 0, st, pmean, pm2, nch, sh.rows_blk, M, C,
                     eps, mean, rstd);
  ps.done_bytes("bn_stats", (double)M * C * (f32 ? 4 : 2));
  PG_LAUNCH_CHECK();
}

// a = [relu]((x - mean[c]) * scale[b][c] + shift[b][c]) stored in the
// activation type: the BN(+ReLU) operand of the next convolution, computed
// once per element instead of once per filter tap.  Padded channels get 0.
// One thread per (pixel, 8 channels): 16-byte loads and stores.
// Block layout of the elementwise BN passes: P = 256 / CC row lanes of CC
// 8-channel groups (a pixel's 16-byte chunks in lane order, so a row lane
// reads whole pixel rows), each thread walking kBnRows rows P apart; the
// per-channel constants stay in registers, the per-image tables are reloaded
// only when a row starts a new image.
constexpr int kBnRows = 4;

template <typename T>
__global__ __launch_bounds__(256) void k_bn_apply(const T* x, int64_t M, int CC, FastDiv fdHW, int C, int Cp,
                                                  const float* mean, const float* scale, const float* shift,
                                                  int tab_stride, int relu, T* out) {
  const int P = 256 / CC;
  const int cg = (int)threadIdx.x % CC, ro = (int)threadIdx.x / CC;
  if (ro >= P) return;
  const int c0 = cg * 8;
  const int64_t r0 = (int64_t)blockIdx.x * P * kBnRows + ro;
  float mu[8], sc[8], sh[8];
  load8f<float>(mean + c0, mu);
  int bcur = -1;
#pragma unroll
  for (int k = 0; k < kBnRows; ++k) {
    const int64_t p = r0 + (int64_t)k * P;
    if (p >= M) break;
    const int b = (int)fdiv((uint32_t)p, fdHW);
    if (b != bcur) {
      const int64_t tb = (int64_t)b * tab_stride;
      load8f<float>(scale + tb + c0, sc);
      load8f<float>(shift + tb + c0, sh);
      bcur = b;
    }
    float v[8];
    load8f<T>(x + p * Cp + c0, v);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      float y = (v[e] - mu[e]) * sc[e] + sh[e];
      if (relu) y = fmaxf(y, 0.f);
      v[e] = c0 + e < C ? y : 0.f;
    }
    store8f<T>(out + p * Cp + c0, v);
  }
}

void bn_apply(hipStream_t st, bool f32, const void* x, int64_t M, int HW, int C, int Cp, const float* mean,
              const float* scale, const float* shift, int tab_stride, bool relu, void* out) {
  const int CC = Cp / 8;
  if (M == 0) return;
  PG_CHECK(Cp % 8 == 0 && CC <= 256 && tab_stride % 8 == 0 && M * CC < (1LL << 31), "bn_apply: shape");
  PG_CHECK(((uintptr_t)mean | (uintptr_t)scale | (uintptr_t)shift) % 16 == 0, "bn_apply: table alignment");
  const FastDiv fdHW = make_fastdiv(HW);
  const int64_t rows_blk = (int64_t)(256 / CC) * kBnRows;
  dim3 g((unsigned)cdiv(M, rows_blk));
  ProfScope ps(st);
  if (f32)
    hipLaunchKernelGGL(k_bn_apply<float>, g, dim3(256), 0, st, (const float*)x, M, CC, fdHW, C, Cp, mean, scale,
                       shift, tab_stride, (int)relu, (float*)out);
  else
    hipLaunchKernelGGL(k_bn_apply<bf16_t>, g, dim3(256), 0, st, (const bf16_t*)x, M, CC, fdHW, C, Cp, mean, scale,
                       shift, tab_stride, (int)relu, (bf16_t*)out);
  ps.done_bytes("bn_apply", 2.0 * M * Cp * (f32 ? 4 : 2));
  PG_LAUNCH_CHECK();
}

// Conditional-BN tables for the conv prologue and the backward pass:
//   gain[b][c] = 1 + cond[b] . Wg[c] / sigma_g,  bias[b][c] = cond[b] . Wb[c] / sigma_b
//   scale[b][c] = gain * rstd[c]   (prologue: (x - mean) * scale + bias)
// Padded channels (c >= C) get zeros.  With cond == nullptr the gains and
// biases are per-channel parameters (plain affine BN, B = 1).
__global__ void k_cbn_tables(const float* cond, int dc, const float* Wg, const float* Wb, const float* sg,
                             const float* sb, const float* gain_p, const float* bias_p,
                             const float* rstd, int B, int C, int Cp, float* gain, float* bias,
                             float* scale) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= B * Cp) return;
  const int b = i / Cp, c = i % Cp;
  float g = 0.f, h = 0.f;
  if (c < C) {
    if (cond) {
      float ag = 0.f, ab = 0.f;
      for (int j = 0; j < dc; ++j) {
        const float cj = cond[(int64_t)b * dc + j];
        ag = fmaf(cj, Wg[(int64_t)c * dc + j], ag);
        ab = fmaf(cj, Wb[(int64_t)c * dc + j], ab);
      }
      g = 1.f + ag / *sg;
      h = ab / *sb;
    } else {
      g = gain_p[c];
      h = bias_p[c];
    }
  }
  gain[i] = g;
  bias[i] = h;
  scale[i] = c < C ? g * rstd[c] : 0.f;
}

// Small fp32 GEMM for the conditional-BN linear maps (B x dc by dc x C and
// their transposes): C[i][j] = sum_k A(i, k) B(k, j) [/ *div] [+ C[i][j]],
// A(i, k) = A[i * sai + k * sak], B(k, j) = B[k * sbk + j * sbj].  32 x 32
// tiles through LDS, k in chunks of 32, fixed summation order.  With a
// split of K (blockIdx.z; part != nullptr) each split writes its raw sums
// to part[z][M][N] and k_gemm_reduce adds them in split order.
__global__ __launch_bounds__(256) void k_gemm_small(int M, int N, int K, const float* A, int64_t sai,
                                                    int64_t sak, const float* Bm, int64_t sbk, int64_t sbj,
                                                    float* Cm, int64_t ldc, const float* div, int acc, int kper,
                                                    float* part) {
  __shared__ float As[32][33], Bs[32][33];
  const int i0 = blockIdx.y * 32, j0 = blockIdx.x * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  const int kb = blockIdx.z * kper, ke = min(K, kb + kper);
  float c[4] = {0.f, 0.f, 0.f, 0.f};
  for (int k0 = kb; k0 < ke; k0 += 32) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int r = ty + 8 * q;
      // the lane index runs along whichever dimension is contiguous
      int ai, ak;
      if (sak == 1) { ai = r; ak = tx; } else { ai = tx; ak = r; }
      As[ai][ak] = (i0 + ai < M && k0 + ak < ke) ? A[(i0 + ai) * sai + (int64_t)(k0 + ak) * sak] : 0.f;
      int bk, bj;
      if (sbj == 1) { bk = r; bj = tx; } else { bk = tx; bj = r; }
      Bs[bk][bj] = (k0 + bk < ke && j0 + bj < N) ? Bm[(int64_t)(k0 + bk) * sbk + (j0 + bj) * sbj] : 0.f;
    }
    __syncthreads();
#pragma unroll 8
    for (int kk = 0; kk < 32; ++kk) {
      const float b = Bs[kk][tx];
#pragma unroll
      for (int q = 0; q < 4; ++q) c[q] = fmaf(As[ty + 8 * q][kk], b, c[q]);
    }
    __syncthreads();
  }
  const int j = j0 + tx;
  if (j >= N) return;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int i = i0 + ty + 8 * q;
    if (i >= M) continue;
    if (part) {
      part[((int64_t)blockIdx.z * M + i) * N + j] = c[q];
      continue;
    }
    float v = div ? c[q] / *div : c[q];
    if (acc) v += Cm[(int64_t)i * ldc + j];
    Cm[(int64_t)i * ldc + j] = v;
  }
}

__global__ void k_gemm_reduce(int M, int N, int splits, const float* part, float* Cm, int64_t ldc,
                              const float* div, int acc) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= (int64_t)M * N) return;
  const int i = (int)(e / N), j = (int)(e - (int64_t)i * N);
  float sum = 0.f;
  for (int z = 0; z < splits; ++z) sum += part[(int64_t)z * M * N + e];
  float v = div ? sum / *div : sum;
  if (acc) v += Cm[(int64_t)i * ldc + j];
  Cm[(int64_t)i * ldc + j] = v;
}

static void gemm_small(hipStream_t st, int M, int N, int K, const float* A, int64_t sai, int64_t sak,
                       const float* Bm, int64_t sbk, int64_t sbj, float* Cm, int64_t ldc, const float* div,
                       bool acc, float* part = nullptr, int splits = 1) {
  if (M <= 0 || N <= 0) return;
  if (!part || splits <= 1) {
    hipLaunchKernelGGL(k_gemm_small, dim3((unsigned)cdiv(N, 32), (unsigned)cdiv(M, 32)), dim3(256), 0, st, M, N, K,
                       A, sai, sak, Bm, sbk, sbj, Cm, ldc, div, (int)acc, K, (float*)nullptr);
    return;
  }
  const int kper = (int)cdiv(cdiv(K, splits), 32) * 32;
  splits = (int)cdiv(K, kper);
  hipLaunchKernelGGL(k_gemm_small, dim3((unsigned)cdiv(N, 32), (unsigned)cdiv(M, 32), (unsigned)splits), dim3(256),
                     0, st, M, N, K, A, sai, sak, Bm, sbk, sbj, Cm, ldc, div, (int)acc, kper, part);
  hipLaunchKernelGGL(k_gemm_reduce, dim3((unsigned)cdiv((int64_t)M * N, 256)), dim3(256), 0, st, M, N, splits, part,
                     Cm, ldc, div, (int)acc);
}

// Both conditional-BN linear maps of one BN in one launch (blockIdx.z: 0
// gain, 1 bias), written as the tables the conv prologue and BN backward use:
//   gain[b][c] = 1 + cond[b] . Wg[c] / sigma_g,  scale = gain * rstd[c],
//   bias[b][c] = cond[b] . Wb[c] / sigma_b,  zeros for c >= C (up to Cp).
// Same 32 x 32 tiling and summation order as k_gemm_small.
__global__ __launch_bounds__(256) void k_cbn_lin(int B, int C, int Cp, int dc, const float* cond, const float* Wg,
                                                 const float* Wb, const float* sg, const float* sb,
                                                 const float* rstd, float* gain, float* bias, float* scale) {
  __shared__ float As[32][33], Bs[32][33];
  const bool isg = blockIdx.z == 0;
  const float* Wm = isg ? Wg : Wb;
  const int i0 = blockIdx.y * 32, j0 = blockIdx.x * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  float c[4] = {0.f, 0.f, 0.f, 0.f};
  for (int k0 = 0; k0 < dc; k0 += 32) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int r = ty + 8 * q;
      As[r][tx] = (i0 + r < B && k0 + tx < dc) ? cond[(int64_t)(i0 + r) * dc + k0 + tx] : 0.f;
      Bs[tx][r] = (k0 + tx < dc && j0 + r < C) ? Wm[(int64_t)(j0 + r) * dc + k0 + tx] : 0.f;
    }
    __syncthreads();
#pragma unroll 8
    for (int kk = 0; kk < 32; ++kk) {
      const float b = Bs[kk][tx];
#pragma unroll
      for (int q = 0; q < 4; ++q) c[q] = fmaf(As[ty + 8 * q][kk], b, c[q]);
    }
    __syncthreads();
  }
  const int j = j0 + tx;
  if (j >= Cp) return;
  const float sig = *(isg ? sg : sb);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int i = i0 + ty + 8 * q;
    if (i >= B) continue;
    const int64_t o = (int64_t)i * Cp + j;
    if (isg) {
      const float g = j < C ? 1.f + c[q] / sig : 0.f;
      gain[o] = g;
      scale[o] = j < C ? g * rstd[j] : 0.f;
    } else {
      bias[o] = j < C ? c[q] / sig : 0.f;
    }
  }
}

void cbn_tables(hipStream_t st, const float* cond, int dc, const float* Wg, const float* Wb,
                const float* sg, const float* sb, const float* gain_p, const float* bias_p,
                const float* rstd, int B, int C, int Cp, float* gain, float* bias, float* scale) {
  if (cond) {
    // gain_raw[b][c] = cond[b] . Wg[c] / sigma_g, bias[b][c] = cond[b] . Wb[c] / sigma_b
    hipLaunchKernelGGL(k_cbn_lin, dim3((unsigned)cdiv(Cp, 32), (unsigned)cdiv(B, 32), 2), dim3(256), 0, st, B, C, Cp,
                       dc, cond, Wg, Wb, sg, sb, rstd, gain, bias, scale);
    PG_LAUNCH_CHECK();
    return;
  }
  hipLaunchKernelGGL(k_cbn_tables, dim3((unsigned)cdiv((int64_t)B * Cp, 256)), dim3(256), 0, st, cond, dc,
                     Wg, Wb, sg, sb, gain_p, bias_p, rstd, B, C, Cp, gain, bias, scale);
  PG_LAUNCH_CHECK();
}

// BN backward, pass 1: per (sample, channel) sums over the sample's pixels of
//   dz = g * [bn(x) > 0]  and  dz * xhat,  xhat = (x - mean) * rstd,
// where g is the gradient of ReLU(BN(x)) (fp32; optionally given at 2x
// resolution and summed over 2x2 -- the upsample's adjoint).  Blocks are
// (chunk of a sample's pixels, sample); a thread owns 8 channels of the
// pixels ro, ro + P, ... of the chunk (16-byte loads), and the P partials
// of each channel combine in order through LDS.
struct BnbShape {
  int CC, P, nchs, rows;   // channel groups, phases, chunks per sample, rows per chunk
};
inline BnbShape bnb_shape(int B, int HW, int C) {
  BnbShape s;
  s.CC = (int)(cpad(C) / 8);
  s.P = std::max(1, 256 / s.CC);
  const int maxch = std::max(1, HW / (s.P * kRowsPerThread));
  s.nchs = std::min(maxch, std::max(1, kMaxChunks / B));
  s.rows = (int)cdiv(HW, s.nchs);
  s.nchs = (int)cdiv(HW, s.rows);
  return s;
}

// 8 fp32 gradient values of pixel r (of HW) of sample b at channel c0, read
// directly or as the 2x2 sum at twice the resolution
PG_DEV void load_g8(const float* g, int g_up2, int64_t m, int b, int r, FastDiv fdW, int H, int W, int Cp, int c0,
                    float* v) {
  if (!g_up2) {
    load8f<float>(g + m * Cp + c0, v);
    return;
  }
  const int h = (int)fdiv((uint32_t)r, fdW), w = r - h * W;
  const int64_t base = (((int64_t)b * 2 * H + 2 * h) * 2 * W + 2 * w) * Cp + c0;
  const int64_t dn = (int64_t)2 * W * Cp;
  float a[8], c[8], d[8];
  load8f<float>(g + base, v);
  load8f<float>(g + base + Cp, a);
  load8f<float>(g + base + dn, c);
  load8f<float>(g + base + dn + Cp, d);
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] = (v[e] + a[e]) + (c[e] + d[e]);
}

template <typename T>
__global__ __launch_bounds__(256) void k_bnb_reduce(const float* g, int g_up2, const T* x, int HW, int H, int W,
                                                    FastDiv fdW, int C, int Cp, const float* mean,
                                                    const float* rstd, const float* gain, const float* bias,
                                                    int tab_stride, BnbShape sh, float* p1, float* p2) {
  __shared__ float s_a[256 * 8], s_b[256 * 8];
  const int b = blockIdx.y;
  const int t = threadIdx.x;
  const int cg = t % sh.CC, ph = t / sh.CC;
  const int c0 = cg * 8;
  const int r0 = blockIdx.x * sh.rows;
  const int r1 = min(r0 + sh.rows, HW);
  float s1[8], s2[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) s1[e] = s2[e] = 0.f;
  if (ph < sh.P) {
    float mu[8], rs[8], ga[8], be[8];
    load8f<float>(mean + c0, mu);
    load8f<float>(rstd + c0, rs);
    load8f<float>(gain + (int64_t)b * tab_stride + c0, ga);
    load8f<float>(bias + (int64_t)b * tab_stride + c0, be);
    auto add = [&](const float* xv, const float* gv) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float xh = (xv[e] - mu[e]) * rs[e];
        const float dz = (ga[e] * xh + be[e] > 0.f) ? gv[e] : 0.f;
        s1[e] += dz;
        s2[e] = fmaf(dz, xh, s2[e]);
      }
    };
    int r = r0 + ph;
    // four rows in flight per thread, accumulated in row order
    for (; r + 3 * sh.P < r1; r += 4 * sh.P) {
      float xv[4][8], gv[4][8];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int ru = r + u * sh.P;
        const int64_t m = (int64_t)b * HW + ru;
        load8f<T>(x + m * Cp + c0, xv[u]);
        load_g8(g, g_up2, m, b, ru, fdW, H, W, Cp, c0, gv[u]);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) add(xv[u], gv[u]);
    }
    for (; r < r1; r += sh.P) {
      const int64_t m = (int64_t)b * HW + r;
      float xv[8], gv[8];
      load8f<T>(x + m * Cp + c0, xv);
      load_g8(g, g_up2, m, b, r, fdW, H, W, Cp, c0, gv);
      add(xv, gv);
    }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    s_a[t * 8 + e] = s1[e];
    s_b[t * 8 + e] = s2[e];
  }
  __syncthreads();
  for (int c = t; c < C; c += 256) {
    const int gi = c >> 3, e = c & 7;
    float a1 = 0.f, a2 = 0.f;
    for (int j = 0; j < sh.P; ++j) {
      a1 += s_a[(j * sh.CC + gi) * 8 + e];
      a2 += s_b[(j * sh.CC + gi) * 8 + e];
    }
    const int64_t o = ((int64_t)b * gridDim.x + blockIdx.x) * C + c;
    p1[o] = a1;
    p2[o] = a2;
  }
}

// pass 2a, per (sample, channel): s1 = sum of the chunk partials of dz,
// s2 = of dz * xhat (fixed order), written over the first chunk's slot;
// per-sample gain / bias gradients when dg_stride != 0.
__global__ void k_bnb_fin1(float* p1, float* p2, int nch, int B, int C, float* dgain, float* dbias,
                           int dg_stride) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (int64_t)B * C) return;
  const int b = (int)(i / C), c = (int)(i - (int64_t)b * C);
  float s1 = 0.f, s2 = 0.f;
  for (int j = 0; j < nch; ++j) {
    const int64_t o = ((int64_t)b * nch + j) * C + c;
    s1 += p1[o];
    s2 += p2[o];
  }
  const int64_t o0 = (int64_t)b * nch * C + c;
  p1[o0] = s1;
  p2[o0] = s2;
  if (dg_stride) {
    dbias[(int64_t)b * dg_stride + c] = s1;
    dgain[(int64_t)b * dg_stride + c] = s2;
  }
}

// pass 2b, per channel: A = sum_b gain*s1 / N, Bc = sum_b gain*s2 / N (and the
// plain-BN gain / bias gradients sum_b s2, sum_b s1); 16 waves stride the
// samples, combined in order.
__global__ __launch_bounds__(1024) void k_bnb_fin2(const float* p1, const float* p2, int nch, int B, int C,
                                                   const float* gain, int tab_stride, int64_t N, float* dgain,
                                                   float* dbias, float* A, float* Bc, int dg_stride) {
  __shared__ float sh[4][16][64];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int c = blockIdx.x * 64 + lane;
  float a = 0.f, bb = 0.f, ab = 0.f, ag = 0.f;
  if (c < C)
    for (int b = wv; b < B; b += 16) {
      const int64_t o0 = (int64_t)b * nch * C + c;
      const float s1 = p1[o0], s2 = p2[o0];
      const float ga = gain[(int64_t)b * tab_stride + c];
      a = fmaf(ga, s1, a);
      bb = fmaf(ga, s2, bb);
      ab += s1;
      ag += s2;
    }
  sh[0][wv][lane] = a; sh[1][wv][lane] = bb; sh[2][wv][lane] = ab; sh[3][wv][lane] = ag;
  __syncthreads();
  if (wv == 0 && c < C) {
    float t[4] = {0.f, 0.f, 0.f, 0.f};
    for (int w = 0; w < 16; ++w)
      for (int q = 0; q < 4; ++q) t[q] += sh[q][w][lane];
    A[c] = t[0] / (float)N;
    Bc[c] = t[1] / (float)N;
    if (!dg_stride) {
      dbias[c] = t[2];
      dgain[c] = t[3];
    }
  }
}

// pass 3: dx = rstd * (gain * dz - A - xhat * Bc) (+ res, at the same pixel),
// in the block layout of k_bn_apply (16-byte loads and stores).
template <typename T>
__global__ __launch_bounds__(256) void k_bnb_apply(const float* g, int g_up2, const T* x, int64_t M, int CC,
                                                   FastDiv fdHW, FastDiv fdW, int HW, int H, int W, int C, int Cp,
                                                   const float* mean, const float* rstd, const float* gain,
                                                   const float* bias, int tab_stride, const float* A,
                                                   const float* Bc, const float* res, T* dx) {
  const int P = 256 / CC;
  const int cg = (int)threadIdx.x % CC, ro = (int)threadIdx.x / CC;
  if (ro >= P) return;
  const int c0 = cg * 8;
  const int64_t r0 = (int64_t)blockIdx.x * P * kBnRows + ro;
  float mu[8], rs[8], aa[8], bb[8], ga[8], be[8];
  load8f<float>(mean + c0, mu);
  load8f<float>(rstd + c0, rs);
  load8f<float>(A + c0, aa);
  load8f<float>(Bc + c0, bb);
  int bcur = -1;
#pragma unroll
  for (int k = 0; k < kBnRows; ++k) {
    const int64_t p = r0 + (int64_t)k * P;
    if (p >= M) break;
    const int b = (int)fdiv((uint32_t)p, fdHW);
    if (b != bcur) {
      load8f<float>(gain + (int64_t)b * tab_stride + c0, ga);
      load8f<float>(bias + (int64_t)b * tab_stride + c0, be);
      bcur = b;
    }
    const int r = (int)(p - (int64_t)b * HW);
    float xv[8], gv[8];
    load8f<T>(x + p * Cp + c0, xv);
    load_g8(g, g_up2, p, b, r, fdW, H, W, Cp, c0, gv);
    float rv[8];
    if (res) load8f<float>(res + p * Cp + c0, rv);
    float out[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float xh = (xv[e] - mu[e]) * rs[e];
      const float dz = (ga[e] * xh + be[e] > 0.f) ? gv[e] : 0.f;
      float o = rs[e] * (ga[e] * dz - aa[e] - xh * bb[e]);
      if (res) o += rv[e];
      out[e] = c0 + e < C ? o : 0.f;
    }
    store8f<T>(dx + p * Cp + c0, out);
  }
}

size_t bn_bwd_ws_bytes(int B, int HW, int C) {
  const BnbShape sh = bnb_shape(B, HW, C);
  return 2 * align256((size_t)B * sh.nchs * C * 4) + 2 * align256((size_t)cpad(C) * 4);
}

void bn_bwd(hipStream_t st, bool f32, const float* g, bool g_up2, const void* x, int B, int H, int W,
            int C, int Cp, const float* mean, const float* rstd, const float* gain, const float* bias,
            int tab_stride, const float* res, void* dx, float* dgain, float* dbias, int dg_stride,
            void* ws) {
  const int HW = H * W;
  const BnbShape sh = bnb_shape(B, HW, C);
  PG_CHECK(Cp % 8 == 0 && Cp >= cpad(C) && tab_stride % 8 == 0, "bn_bwd: channel layout");
  PG_CHECK(((uintptr_t)mean | (uintptr_t)rstd | (uintptr_t)gain | (uintptr_t)bias | (uintptr_t)g) % 16 == 0,
           "bn_bwd: alignment");
  const int nch = sh.nchs;
  float* p1 = (float*)ws;
  float* p2 = (float*)((char*)p1 + align256((size_t)B * nch * C * 4));
  float* A = (float*)((char*)p2 + align256((size_t)B * nch * C * 4));
  float* Bc = (float*)((char*)A + align256((size_t)cpad(C) * 4));
  const FastDiv fdW = make_fastdiv(W);
  dim3 g1(nch, B);
  // algorithmic bytes: x and the fp32 output gradient (at its own
  // resolution) read for the statistics, then again with dx written
  const double gbytes = 4.0 * (double)B * HW * C / (g_up2 ? 4 : 1), xbytes = (double)B * HW * Cp * (f32 ? 4 : 2);
  ProfScope ps(st);
  if (f32)
    hipLaunchKernelGGL(k_bnb_reduce<float>, g1, dim3(256), 0, st, g, (int)g_up2, (const float*)x, HW, H, W, fdW,
                       C, Cp, mean, rstd, gain, bias, tab_stride, sh, p1, p2);
  else
    hipLaunchKernelGGL(k_bnb_reduce<bf16_t>, g1, dim3(256), 0, st, g, (int)g_up2, (const bf16_t*)x, HW, H, W, fdW,
                       C, Cp, mean, rstd, gain, bias, tab_stride, sh, p1, p2);
  hipLaunchKernelGGL(k_bnb_fin1, dim3((unsigned)cdiv((int64_t)B * C, 256)), dim3(256), 0, st, p1, p2, nch, B, C,
                     dgain, dbias, dg_stride);
  hipLaunchKernelGGL(k_bnb_fin2, dim3((unsigned)cdiv(C, 64)), dim3(1024), 0, st, p1, p2, nch, B, C, gain,
                     tab_stride, (int64_t)B * HW, dgain, dbias, A, Bc, dg_stride);
  ps.done_bytes("bn_bwd_stats", gbytes + xbytes);
  const int64_t M = (int64_t)B * HW;
  const int CC = Cp / 8;
  PG_CHECK(M * CC < (1LL << 31) && M < (1LL << 31) && CC <= 256, "bn_bwd: too large");
  dim3 g3((unsigned)cdiv(M, (int64_t)(256 / CC) * kBnRows));
  const FastDiv fdHW = make_fastdiv(HW);
  ProfScope ps2(st);
  if (f32)
    hipLaunchKernelGGL(k_bnb_apply<float>, g3, dim3(256), 0, st, g, (int)g_up2, (const float*)x, M, CC, fdHW, fdW,
                       HW, H, W, C, Cp, mean, rstd, gain, bias, tab_stride, A, Bc, res, (float*)dx);
  else
    hipLaunchKernelGGL(k_bnb_apply<bf16_t>, g3, dim3(256), 0, st, g, (int)g_up2, (const bf16_t*)x, M, CC, fdHW,
                       fdW, HW, H, W, C, Cp, mean, rstd, gain, bias, tab_stride, A, Bc, res, (bf16_t*)dx);
  ps2.done_bytes("bn_bwd_apply", gbytes + 2.0 * xbytes + (res ? 4.0 * (double)M * C : 0.0));
  PG_LAUNCH_CHECK();
}

// Linear-map gradients of the conditional BN:
//   dW[c][j] = sum_b dgb[b][c] cond[b][j]   (gradient of W/sigma; SN bwd follows)
//   dcond[b][j] (+)= sum_c dgb[b][c] W[c][j] / sigma
size_t cbn_linear_bwd_ws_bytes(int B, int dc) { return align256((size_t)kLinSplits * B * dc * 4); }

void cbn_linear_bwd(hipStream_t st, const float* dgb, int B, int C, int Cp, const float* cond, int dc,
                    const float* W, const float* sigma, float* dW, float* dcond, bool accumulate, float* ws) {
  // dW[c][j] = sum_b dgb[b][c] cond[b][j];  dcond[b][j] (+)= sum_c dgb[b][c] W[c][j] / sigma
  gemm_small(st, C, dc, B, dgb, 1, Cp, cond, dc, 1, dW, dc, nullptr, false);
  // K = C is long and M x N = B x dc small: split K for parallelism
  const int splits = ws ? (int)std::min<int64_t>(kLinSplits, cdiv(C, 128)) : 1;
  gemm_small(st, B, dc, C, dgb, Cp, 1, W, dc, 1, dcond, dc, sigma, accumulate, ws, splits);
  PG_LAUNCH_CHECK();
}

// 2x2 average pool, 8 channels per thread
template <typename T>
__global__ __launch_bounds__(256) void k_avgpool2(const T* x, int64_t n8, int CC, FastDiv fdCC, FastDiv fdWo,
                                                  int Ho, int Wo, T* out) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n8) return;
  const int p = (int)fdiv((uint32_t)i, fdCC);
  const int cc = (int)i - p * CC;
  const int t = (int)fdiv((uint32_t)p, fdWo);
  const int j = p - t * Wo;           // t = b * Ho + i
  const int64_t W2 = 2LL * Wo;
  const int64_t r0 = (2LL * t) * W2 + 2 * j;   // (b, 2i, 2j) as a pixel of the input
  const int64_t Cp = (int64_t)CC * 8;
  float a[8], v[8];
  load8f<T>(x + r0 * Cp + cc * 8, a);
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] = a[e];
  load8f<T>(x + (r0 + 1) * Cp + cc * 8, a);
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] += a[e];
  load8f<T>(x + (r0 + W2) * Cp + cc * 8, a);
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] += a[e];
  load8f<T>(x + (r0 + W2 + 1) * Cp + cc * 8, a);
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] = (v[e] + a[e]) * 0.25f;
  (void)Ho;
  store8f<T>(out + i * 8, v);
}

void avgpool2(hipStream_t st, bool f32, const void* x, int B, int H, int W, int Cp, void* out) {
  PG_CHECK(H % 2 == 0 && W % 2 == 0 && Cp % 8 == 0, "avgpool2: shape");
  const int Ho = H / 2, Wo = W / 2, CC = Cp / 8;
  const int64_t n8 = (int64_t)B * Ho * Wo * CC;
  if (n8 == 0) return;
  PG_CHECK(n8 < (1LL << 31), "avgpool2: size");
  const FastDiv fdCC = make_fastdiv(CC), fdWo = make_fastdiv(Wo);
  dim3 g((unsigned)cdiv(n8, 256));
  ProfScope ps(st);
  if (f32)
    hipLaunchKernelGGL(k_avgpool2<float>, g, dim3(256), 0, st, (const float*)x, n8, CC, fdCC, fdWo, Ho, Wo,
                       (float*)out);
  else
    hipLaunchKernelGGL(k_avgpool2<bf16_t>, g, dim3(256), 0, st, (const bf16_t*)x, n8, CC, fdCC, fdWo, Ho, Wo,
                       (bf16_t*)out);
  ps.done_bytes("avgpool2", 5.0 * 8.0 * n8 * (f32 ? 4 : 2));
  PG_LAUNCH_CHECK();
}

// elementwise helpers
__global__ void k_fill(float* p, int64_t n, float v) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) p[i] = v;
}
void fill(hipStream_t st, float* p, int64_t n, float v) {
  if (n <= 0) return;
  hipLaunchKernelGGL(k_fill, dim3((unsigned)cdiv(n, 256)), dim3(256), 0, st, p, n, v);
  PG_LAUNCH_CHECK();
}

}  // namespace pg
