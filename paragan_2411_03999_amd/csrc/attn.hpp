// Launchers of the self-attention kernels (attention.hip).
#pragma once
#include "misc.hpp"

namespace pg {

struct AttnDims {
  int B, H, W, HW, L, Lp, HWp;
  int dk, dv, Nqkv;   // padded query/key width (32), value width, fused projection width
};

void attn_pool(hipStream_t st, const AttnDims& a, const void* qkv, void* kp, void* vp);
// lse2: log2-sum-exp2 per query, [B][HWp] (+inf for padded queries)
// o: bf16 [B][HW][dv]; o32: the same rows in fp32 (for the backward)
void attn_fwd_core(hipStream_t st, const AttnDims& a, const void* qkv, const void* kp, const void* vp, void* o,
                   float* o32, float* lse2);
// o32: the forward's fp32 output [B][HW][dv], for the softmax backward's row term dO . o
void attn_bwd_core(hipStream_t st, const AttnDims& a, const void* qkv, const void* dO, const float* o32,
                   const void* kp, const void* vp, const float* lse2, float* Dv, void* dk, void* dvv, void* dqkv);
void attn_dgamma(hipStream_t st, const void* wo, const float* dwo, int64_t n, float* out);

}  // namespace pg
