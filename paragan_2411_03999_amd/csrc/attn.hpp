// Launchers of the self-attention kernels (attention.hip).
#pragma once
#include "misc.hpp"

namespace pg {

struct AttnDims {
  int B, H, W, HW, L, Lp, HWp;
  int dk, dv, Nqkv;   // padded query/key width (32), value width, fused projection width
};

void attn_pool(hipStream_t st, const AttnDims& a, const void* qkv, void* kp, void* kt, void* vp, void* vt);
void attn_transpose(hipStream_t st, const AttnDims& a, const void* src, int ld, int c0, int C, void* dst);
void attn_fwd_core(hipStream_t st, const AttnDims& a, const void* qkv, const void* kp, const void* vt, void* o,
                   float* lse);
void attn_bwd_core(hipStream_t st, const AttnDims& a, const void* qkv, const void* o, const void* dO,
                   const void* kp, const void* kt, const void* vp, const void* qt, const void* dOt,
                   const float* lse, float* Dv, void* dk, void* dvv, void* dqkv);
void attn_dgamma(hipStream_t st, const void* wo, const float* dwo, int64_t n, float* out);

}  // namespace pg
