// Gating (Alg. 7: scores, softmax, TopKIndices, w = p[I]) and its adjoint on the data owner.
//
// Scores are accumulated in fp64 from the exact products of the stored inputs and rounded once
// to fp32, so the top-k decision is reproducible from the inputs alone. Selection happens at
// wavefront level: k rounds of a 64-lane butterfly argmax on (score, -expert index).
#include "pcmoe_internal.h"
#include <math.h>

namespace pcmoe {

constexpr int RT_TOK = 64;  // tokens per block
constexpr int RT_DC = 64;   // d-columns staged in LDS per step
constexpr int RT_PITCH = RT_DC + 1;

// NE = experts per thread (16 expert lanes per block): E <= 16*NE.
template <typename T, int NE>
__global__ __launch_bounds__(256) void route_fwd_kernel(const T* __restrict__ x, const T* __restrict__ wr,
                                                        const float* __restrict__ bias, int bias_div, int Tn,
                                                        int d, int E, int k, int renorm,
                                                        float* __restrict__ logits, int32_t* __restrict__ idx,
                                                        float* __restrict__ gw) {
  extern __shared__ float sm[];
  float* xs = sm;                       // [64][65]
  float* wsm = sm + RT_TOK * RT_PITCH;  // [E][65]
  const int tid = threadIdx.x;
  const int t0 = blockIdx.x * RT_TOK;
  const int tt = tid & 15, te = tid >> 4;

  double acc[4][NE];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < NE; ++b) acc[a][b] = 0.0;

  for (int k0 = 0; k0 < d; k0 += RT_DC) {
    __syncthreads();
    for (int i = tid; i < RT_TOK * RT_DC; i += 256) {
      int r = i / RT_DC, c = i % RT_DC, t = t0 + r;
      xs[r * RT_PITCH + c] = (t < Tn) ? to_f(x[(size_t)t * d + k0 + c]) : 0.f;
    }
    for (int i = tid; i < E * RT_DC; i += 256) {
      int r = i / RT_DC, c = i % RT_DC;
      wsm[r * RT_PITCH + c] = to_f(wr[(size_t)r * d + k0 + c]);
    }
    __syncthreads();
#pragma unroll 4
    for (int c = 0; c < RT_DC; ++c) {
      double xv[4];
#pragma unroll
      for (int a = 0; a < 4; ++a) xv[a] = (double)xs[(tt + 16 * a) * RT_PITCH + c];
#pragma unroll
      for (int b = 0; b < NE; ++b) {
        int e = te + 16 * b;
        double wv = (e < E) ? (double)wsm[e * RT_PITCH + c] : 0.0;
#pragma unroll
        for (int a = 0; a < 4; ++a) acc[a][b] = fma(xv[a], wv, acc[a][b]);
      }
    }
  }
  __syncthreads();
  // scores (+ bias) rounded once to fp32; keep the block's tile in LDS for the selection
  float* lsm = sm;  // [64][E+1]
  const int lp = E + 1;
#pragma unroll
  for (int a = 0; a < 4; ++a) {
    int r = tt + 16 * a, t = t0 + r;
#pragma unroll
    for (int b = 0; b < NE; ++b) {
      int e = te + 16 * b;
      if (t < Tn && e < E) {
        double v = acc[a][b];
        if (bias) v += (double)bias[(size_t)(t / bias_div) * E + e];
        float L = (float)v;
        logits[(size_t)t * E + e] = L;
        lsm[r * lp + e] = L;
      }
    }
  }
  __syncthreads();

  const int lane = tid & 63, wave = tid >> 6;
  for (int r = wave; r < RT_TOK; r += 4) {
    const int t = t0 + r;
    if (t >= Tn) break;
    float v[4];
    bool taken[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      int e = lane + 64 * q;
      v[q] = (e < E) ? lsm[r * lp + e] : -INFINITY;
      taken[q] = (e >= E);
    }
    float myv = -INFINITY;
    int myi = 0;
    for (int j = 0; j < k; ++j) {
      float bv = -INFINITY;
      int bi = 0x7fffffff;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        int e = lane + 64 * q;
        if (!taken[q] && (v[q] > bv || (v[q] == bv && e < bi))) {
          bv = v[q];
          bi = e;
        }
      }
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) {
        float ov = __shfl_xor(bv, off, 64);
        int oi = __shfl_xor(bi, off, 64);
        if (ov > bv || (ov == bv && oi < bi)) {
          bv = ov;
          bi = oi;
        }
      }
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (lane + 64 * q == bi) taken[q] = true;
      if (lane == j) {
        myv = bv;
        myi = bi;
      }
    }
    const float m = __shfl(myv, 0, 64);  // the largest score of the token
    float ex = (lane < k) ? expf(myv - m) : 0.f;
    float Z;
    if (renorm) {
      Z = wave_sum(ex);
    } else {
      float part = 0.f;
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (lane + 64 * q < E) part += expf(v[q] - m);
      Z = wave_sum(part);
    }
    if (lane < k) {
      idx[(size_t)t * k + lane] = myi;
      gw[(size_t)t * k + lane] = ex / Z;
    }
  }
}

template <typename T>
static hipError_t route_fwd_t(const moe_desc& d, const void* x, const void* wr, const float* bias, int bg,
                              float* logits, int32_t* idx, float* w, hipStream_t s) {
  const int E = d.n_experts;
  dim3 grid((d.T + RT_TOK - 1) / RT_TOK);
  size_t lds_a = (size_t)(RT_TOK + E) * RT_PITCH * sizeof(float);
  size_t lds_b = (size_t)RT_TOK * (E + 1) * sizeof(float);
  size_t lds = lds_a > lds_b ? lds_a : lds_b;
  int div = d.T / (bg > 0 ? bg : 1);
  KernelTimer kt("route_fwd", s);
#define RT_LAUNCH(NE)                                                                                            \
  do {                                                                                                           \
    if (lds > 65536) {                                                                                           \
      hipError_t e_ = hipFuncSetAttribute((const void*)route_fwd_kernel<T, NE>,                                   \
                                          hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);                 \
      if (e_ != hipSuccess) return e_;                                                                           \
    }                                                                                                            \
    hipLaunchKernelGGL((route_fwd_kernel<T, NE>), grid, dim3(256), lds, s, (const T*)x, (const T*)wr, bias, div, \
                       d.T, d.d_model, E, d.top_k, d.renormalize, logits, idx, w);                               \
  } while (0)
  if (E <= 16) RT_LAUNCH(1);
  else if (E <= 64) RT_LAUNCH(4);
  else RT_LAUNCH(16);
#undef RT_LAUNCH
  return hipGetLastError();
}

hipError_t launch_route_fwd(const moe_desc& d, const void* x, const void* wr, const float* bias, int bg,
                            float* logits, int32_t* idx, float* w, hipStream_t s) {
  if (d.dtype == MOE_BF16) return route_fwd_t<bf16>(d, x, wr, bias, bg, logits, idx, w, s);
  return route_fwd_t<float>(d, x, wr, bias, bg, logits, idx, w, s);
}

// ------------------------------------------------------------------------------ backward

// dscores per token (one wavefront per token).
__global__ __launch_bounds__(256) void route_dlogits_kernel(int Tn, int E, int k, int renorm,
                                                            const float* __restrict__ logits,
                                                            const int32_t* __restrict__ idx,
                                                            const float* __restrict__ gw,
                                                            const float* __restrict__ dgate,
                                                            float* __restrict__ dl) {
  const int lane = threadIdx.x & 63;
  const int wave = (blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int nwaves = (gridDim.x * blockDim.x) >> 6;
  for (int t = wave; t < Tn; t += nwaves) {
    float wj = 0.f, gj = 0.f;
    int ij = -1;
    if (lane < k) {
      wj = gw[(size_t)t * k + lane];
      gj = dgate[(size_t)t * k + lane];
      ij = idx[(size_t)t * k + lane];
    }
    if (renorm) {
      const float sgw = wave_sum(wj * gj);
      for (int e0 = 0; e0 < E; e0 += 64) {
        int e = e0 + lane;
        float val = 0.f;
        for (int jj = 0; jj < k; ++jj) {
          int i2 = __shfl(ij, jj, 64);
          float w2 = __shfl(wj, jj, 64), g2 = __shfl(gj, jj, 64);
          if (e == i2) val = w2 * (g2 - sgw);
        }
        if (e < E) dl[(size_t)t * E + e] = val;
      }
    } else {
      // p over all E experts; g = dgate scattered onto E
      float M = -INFINITY;
      for (int e = lane; e < E; e += 64) M = fmaxf(M, logits[(size_t)t * E + e]);
      M = wave_max(M);
      float zp = 0.f;
      for (int e = lane; e < E; e += 64) zp += expf(logits[(size_t)t * E + e] - M);
      const float Z = wave_sum(zp);
      float spg = 0.f;
      for (int e0 = 0; e0 < E; e0 += 64) {
        int e = e0 + lane;
        float g = 0.f;
        for (int jj = 0; jj < k; ++jj) {
          int i2 = __shfl(ij, jj, 64);
          float g2 = __shfl(gj, jj, 64);
          if (e == i2) g = g2;
        }
        float p = (e < E) ? expf(logits[(size_t)t * E + e] - M) / Z : 0.f;
        spg += p * g;
      }
      const float S = wave_sum(spg);
      for (int e0 = 0; e0 < E; e0 += 64) {
        int e = e0 + lane;
        float p = 0.f, g = 0.f;
        if (e < E) p = expf(logits[(size_t)t * E + e] - M) / Z;
        for (int jj = 0; jj < k; ++jj) {
          int i2 = __shfl(ij, jj, 64);
          float g2 = __shfl(gj, jj, 64);
          if (e == i2) g = g2;
        }
        if (e < E) dl[(size_t)t * E + e] = p * (g - S);
      }
    }
  }
}

// Partial dW_router over one chunk of tokens: part[chunk][e][c] = sum_{t in chunk} dl[t][e] * x[t][c].
constexpr int RB_TOK = 64;
template <typename T, int NE4>
__global__ __launch_bounds__(256) void route_dw_partial_kernel(int Tn, int d, int E, int tok_per_chunk,
                                                               const T* __restrict__ x,
                                                               const float* __restrict__ dl,
                                                               float* __restrict__ part) {
  extern __shared__ float dls[];  // [RB_TOK][E]
  const int tid = threadIdx.x;
  const int c = blockIdx.x * 64 + (tid & 63);
  const int er = tid >> 6;
  const int chunk = blockIdx.y;
  const int tb = chunk * tok_per_chunk;
  const int te = min(Tn, tb + tok_per_chunk);
  float acc[NE4];
#pragma unroll
  for (int b = 0; b < NE4; ++b) acc[b] = 0.f;
  for (int s0 = tb; s0 < te; s0 += RB_TOK) {
    const int n = min(RB_TOK, te - s0);
    __syncthreads();
    for (int i = tid; i < n * E; i += 256) dls[i] = dl[(size_t)s0 * E + i];
    __syncthreads();
    for (int r = 0; r < n; ++r) {
      float xv = to_f(x[(size_t)(s0 + r) * d + c]);
#pragma unroll
      for (int b = 0; b < NE4; ++b) {
        int e = er + 4 * b;
        if (e < E) acc[b] = fmaf(dls[r * E + e], xv, acc[b]);
      }
    }
  }
#pragma unroll
  for (int b = 0; b < NE4; ++b) {
    int e = er + 4 * b;
    if (e < E) part[((size_t)chunk * E + e) * d + c] = acc[b];
  }
}

__global__ __launch_bounds__(256) void route_dw_reduce_kernel(int n, int nchunks, const float* __restrict__ part,
                                                              float* __restrict__ out) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) {
    float s = 0.f;
    for (int c = 0; c < nchunks; ++c) s += part[(size_t)c * n + i];
    out[i] = s;
  }
}

static void route_bwd_chunks(const moe_desc& d, int* nch, int* tpc) {
  int ncol = d.d_model / 64;
  int maxch = (d.T + RB_TOK - 1) / RB_TOK;
  int want = (1024 + ncol - 1) / ncol;
  int n = want < maxch ? want : maxch;
  if (n < 1) n = 1;
  int per = (d.T + n - 1) / n;
  per = ((per + RB_TOK - 1) / RB_TOK) * RB_TOK;
  *tpc = per;
  *nch = (d.T + per - 1) / per;
}

size_t route_bwd_ws_bytes(const moe_desc& d) {
  int nch, tpc;
  route_bwd_chunks(d, &nch, &tpc);
  return align256((size_t)nch * d.n_experts * d.d_model * sizeof(float));
}

template <typename T>
static hipError_t route_bwd_t(const moe_desc& d, const void* x, const float* logits, const int32_t* idx,
                              const float* w, const float* dgate, float* dl, float* dwr, void* ws,
                              hipStream_t s) {
  const int E = d.n_experts;
  {
    KernelTimer kt("route_dlogits", s);
    int blocks = (d.T + 3) / 4;
    if (blocks > 4096) blocks = 4096;
    hipLaunchKernelGGL(route_dlogits_kernel, dim3(blocks), dim3(256), 0, s, d.T, E, d.top_k, d.renormalize,
                       logits, idx, w, dgate, dl);
  }
  int nch, tpc;
  route_bwd_chunks(d, &nch, &tpc);
  float* part = (float*)ws;
  {
    KernelTimer kt("route_dw_partial", s);
    dim3 grid(d.d_model / 64, nch);
    size_t lds = (size_t)RB_TOK * E * sizeof(float);  // at most 64 KiB (E <= 256)
#define RB_LAUNCH(NE4)                                                                                        \
  hipLaunchKernelGGL((route_dw_partial_kernel<T, NE4>), grid, dim3(256), lds, s, d.T, d.d_model, E, tpc, \
                     (const T*)x, dl, part)
    if (E <= 8) RB_LAUNCH(2);
    else if (E <= 16) RB_LAUNCH(4);
    else if (E <= 64) RB_LAUNCH(16);
    else RB_LAUNCH(64);
#undef RB_LAUNCH
  }
  {
    KernelTimer kt("route_dw_reduce", s);
    int n = E * d.d_model;
    int blocks = (n + 255) / 256;
    if (blocks > 2048) blocks = 2048;
    hipLaunchKernelGGL(route_dw_reduce_kernel, dim3(blocks), dim3(256), 0, s, n, nch, part, dwr);
  }
  return hipGetLastError();
}

hipError_t launch_route_bwd(const moe_desc& d, const void* x, const float* logits, const int32_t* idx,
                            const float* w, const float* dgate, float* dl, float* dwr, void* ws, hipStream_t s) {
  if (d.dtype == MOE_BF16) return route_bwd_t<bf16>(d, x, logits, idx, w, dgate, dl, dwr, ws, s);
  return route_bwd_t<float>(d, x, logits, idx, w, dgate, dl, dwr, ws, s);
}

}  // namespace pcmoe
