// Expert parameter update (the step that closes the host's expert pass in Alg. 6): SGD or AdamW with decoupled weight
// decay, elementwise in fp32 over the hosted and shared experts' w_gate, w_up and w_down.
// Bandwidth-bound: each thread updates 8 consecutive parameters with 16-byte vector accesses.
#include "pcmoe_internal.h"

#include <math.h>

namespace pcmoe {

struct UpdateArgs {
  void* w[3];             // w_gate, w_up, w_down (dtype)
  const void* g[3];       // their gradients (dtype)
  long n;                 // parameters per tensor
  float* master;          // fp32 [3n] or null
  float* m;               // fp32 [3n] (AdamW)
  float* v;               // fp32 [3n] (AdamW)
  float lr, wd, beta1, beta2, eps;
  float step_size;        // lr / (1 - beta1^t)
  float inv_sqrt_bc2;     // 1 / sqrt(1 - beta2^t)
  float decay;            // 1 - lr * wd
};

// One thread per group of 8 consecutive parameters (measured faster than a grid-stride loop over a
// capped grid).
template <typename T, bool ADAM, bool MASTER>
__global__ __launch_bounds__(256) void expert_update_kernel(UpdateArgs a) {
  constexpr int EP = EPC<T>::value;  // elements per 16-byte chunk of the dtype
  const long per = a.n / 8;          // 8-parameter groups per tensor
  const long q = blockIdx.x * (long)blockDim.x + threadIdx.x;
  if (q < 3 * per) {
    const int seg = (int)(q / per);
    const long e0 = (q - seg * per) * 8;  // first parameter within the tensor
    const long f0 = seg * a.n + e0;       // and within the fp32 state arrays
    T* w = reinterpret_cast<T*>(a.w[seg]) + e0;
    const T* g = reinterpret_cast<const T*>(a.g[seg]) + e0;
    float p[8], gr[8];
#pragma unroll
    for (int c = 0; c < 8 / EP; ++c) chunk_to_f<T>(ld_chunk(g + c * EP), gr + c * EP);
    if (MASTER) {
      chunk_to_f<float>(ld_chunk(a.master + f0), p);
      chunk_to_f<float>(ld_chunk(a.master + f0 + 4), p + 4);
    } else {
#pragma unroll
      for (int c = 0; c < 8 / EP; ++c) chunk_to_f<T>(ld_chunk(w + c * EP), p + c * EP);
    }
    if (ADAM) {
      float mm[8], vv[8];
      chunk_to_f<float>(ld_chunk(a.m + f0), mm);
      chunk_to_f<float>(ld_chunk(a.m + f0 + 4), mm + 4);
      chunk_to_f<float>(ld_chunk(a.v + f0), vv);
      chunk_to_f<float>(ld_chunk(a.v + f0 + 4), vv + 4);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        p[i] *= a.decay;
        mm[i] = a.beta1 * mm[i] + (1.f - a.beta1) * gr[i];
        vv[i] = a.beta2 * vv[i] + (1.f - a.beta2) * gr[i] * gr[i];
        p[i] -= a.step_size * mm[i] / (sqrtf(vv[i]) * a.inv_sqrt_bc2 + a.eps);
      }
      st_chunk(a.m + f0, f_to_chunk<float>(mm));
      st_chunk(a.m + f0 + 4, f_to_chunk<float>(mm + 4));
      st_chunk(a.v + f0, f_to_chunk<float>(vv));
      st_chunk(a.v + f0 + 4, f_to_chunk<float>(vv + 4));
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) p[i] -= a.lr * (gr[i] + a.wd * p[i]);
    }
    if (MASTER) {
      st_chunk(a.master + f0, f_to_chunk<float>(p));
      st_chunk(a.master + f0 + 4, f_to_chunk<float>(p + 4));
    }
#pragma unroll
    for (int c = 0; c < 8 / EP; ++c) st_chunk(w + c * EP, f_to_chunk<T>(p + c * EP));
  }
}

hipError_t launch_expert_update(const moe_desc& d, const moe_opt& o, void* wg, void* wu, void* wd, const void* gg,
                                const void* gu, const void* gd, float* master, float* m, float* v,
                                hipStream_t s) {
  UpdateArgs a;
  a.w[0] = wg; a.w[1] = wu; a.w[2] = wd;
  a.g[0] = gg; a.g[1] = gu; a.g[2] = gd;
  a.n = (long)(d.local_count + d.n_shared) * d.d_ff * d.d_model;
  a.master = master; a.m = m; a.v = v;
  a.lr = o.lr; a.wd = o.weight_decay; a.beta1 = o.beta1; a.beta2 = o.beta2; a.eps = o.eps;
  const double bc1 = 1.0 - pow((double)o.beta1, (double)o.step);
  const double bc2 = 1.0 - pow((double)o.beta2, (double)o.step);
  a.step_size = o.kind == MOE_OPT_ADAMW ? (float)((double)o.lr / bc1) : 0.f;
  a.inv_sqrt_bc2 = o.kind == MOE_OPT_ADAMW ? (float)(1.0 / sqrt(bc2)) : 0.f;
  a.decay = (float)(1.0 - (double)o.lr * (double)o.weight_decay);
  const long groups = 3 * (a.n / 8);
  const long blocks = (groups + 255) / 256;  // < 2^31 (checked by moe_expert_update)
  KernelTimer kt("expert_update", s);
#define UPD(T, ADAM, MASTER) \
  hipLaunchKernelGGL((expert_update_kernel<T, ADAM, MASTER>), dim3((unsigned)blocks), dim3(256), 0, s, a)
  const bool adam = o.kind == MOE_OPT_ADAMW, mst = master != nullptr;
  if (d.dtype == MOE_BF16) {
    if (adam) { if (mst) UPD(bf16, true, true); else UPD(bf16, true, false); }
    else { if (mst) UPD(bf16, false, true); else UPD(bf16, false, false); }
  } else {
    if (adam) { if (mst) UPD(float, true, true); else UPD(float, true, false); }
    else { if (mst) UPD(float, false, true); else UPD(float, false, false); }
  }
#undef UPD
  return hipGetLastError();
}

}  // namespace pcmoe
