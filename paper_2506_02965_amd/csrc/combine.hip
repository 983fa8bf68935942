// Owner-side combine of Alg. 3 (y_t = sum over the token's selected experts of w * output, plus
// the always-active shared experts) and its adjoint (Alg. 5 / Sec. 3.2: each host receives the
// gradient w.r.t. its expert's output, w * dY; the owner keeps dgate = <dY, output>).
// One wavefront per token; 16-byte chunks along d; fp32 sums in slot order, then shared experts.
#include "pcmoe_internal.h"

namespace pcmoe {

static int token_blocks(int Tn) {
  int b = (Tn + 3) / 4;
  return b > 8192 ? 8192 : (b < 1 ? 1 : b);
}

// Each lane handles CPL 16-byte chunks per pass; the chunks of all KM slots and of up to SM shared experts are
// loaded together (one round trip per token for its map and weights, one per pass for its rows); shared
// experts beyond SM are added one at a time after them. Sums: slots j in order, then shared experts in order.
template <typename T, int KM, int SM>
__global__ __launch_bounds__(256) void combine_kernel(int Tn, int k, int S, int cpr, const Chunk* __restrict__ yp,
                                                      const int32_t* __restrict__ s2r,
                                                      const float* __restrict__ gw, Chunk* __restrict__ y) {
  constexpr int N = EPC<T>::value;
  constexpr int CPL = chunks_per_lane(KM + SM);
  const int lane = threadIdx.x & 63;
  const int wave = (blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int nwaves = (gridDim.x * blockDim.x) >> 6;
  const size_t shared_base = (size_t)Tn * k;
  for (int t = wave; t < Tn; t += nwaves) {
    int rows[KM];
    float w[KM];
#pragma unroll
    for (int j = 0; j < KM; ++j) {
      rows[j] = (j < k) ? s2r[(size_t)t * k + j] : -1;
      w[j] = (j < k) ? gw[(size_t)t * k + j] : 0.f;
    }
    for (int c0 = lane; c0 < cpr; c0 += 64 * CPL) {
      Chunk in[KM][CPL], sh[SM > 0 ? SM : 1][CPL];
#pragma unroll
      for (int j = 0; j < KM; ++j)
#pragma unroll
        for (int u = 0; u < CPL; ++u)
          in[j][u] = (rows[j] >= 0 && c0 + 64 * u < cpr) ? yp[(size_t)rows[j] * cpr + c0 + 64 * u] : zero_chunk();
#pragma unroll
      for (int s = 0; s < SM; ++s)
#pragma unroll
        for (int u = 0; u < CPL; ++u)
          sh[s][u] = (c0 + 64 * u < cpr) ? yp[(shared_base + (size_t)s * Tn + t) * cpr + c0 + 64 * u] : zero_chunk();
#pragma unroll
      for (int u = 0; u < CPL; ++u) {
        const int c = c0 + 64 * u;
        float acc[N], v[N];
#pragma unroll
        for (int i = 0; i < N; ++i) acc[i] = 0.f;
#pragma unroll
        for (int j = 0; j < KM; ++j) {
          if (rows[j] >= 0) {
            chunk_to_f<T>(in[j][u], v);
#pragma unroll
            for (int i = 0; i < N; ++i) acc[i] = fmaf(w[j], v[i], acc[i]);
          }
        }
#pragma unroll
        for (int s = 0; s < SM; ++s) {
          chunk_to_f<T>(sh[s][u], v);
#pragma unroll
          for (int i = 0; i < N; ++i) acc[i] += v[i];
        }
        if (c < cpr) {
          for (int s = SM; s < S; ++s) {
            chunk_to_f<T>(yp[(shared_base + (size_t)s * Tn + t) * cpr + c], v);
#pragma unroll
            for (int i = 0; i < N; ++i) acc[i] += v[i];
          }
          y[(size_t)t * cpr + c] = f_to_chunk<T>(acc);
        }
      }
    }
  }
}

template <typename T, int KM, int CPL>
__global__ __launch_bounds__(256) void combine_bwd_kernel(int Tn, int k, int cpr, const Chunk* __restrict__ dy,
                                                          const Chunk* __restrict__ yp,
                                                          const int32_t* __restrict__ s2r,
                                                          const float* __restrict__ gw, Chunk* __restrict__ dyp,
                                                          float* __restrict__ dgate) {
  constexpr int N = EPC<T>::value;
  const int lane = threadIdx.x & 63;
  const int wave = (blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int nwaves = (gridDim.x * blockDim.x) >> 6;
  for (int t = wave; t < Tn; t += nwaves) {
    int rows[KM];
    float w[KM], dot[KM];
#pragma unroll
    for (int j = 0; j < KM; ++j) {
      rows[j] = (j < k) ? s2r[(size_t)t * k + j] : -1;
      w[j] = (j < k) ? gw[(size_t)t * k + j] : 0.f;
      dot[j] = 0.f;
    }
    for (int c0 = lane; c0 < cpr; c0 += 64 * CPL) {
      Chunk gc[CPL], in[KM][CPL];
#pragma unroll
      for (int u = 0; u < CPL; ++u) gc[u] = (c0 + 64 * u < cpr) ? dy[(size_t)t * cpr + c0 + 64 * u] : zero_chunk();
#pragma unroll
      for (int j = 0; j < KM; ++j)
#pragma unroll
        for (int u = 0; u < CPL; ++u)
          in[j][u] = (rows[j] >= 0 && c0 + 64 * u < cpr) ? yp[(size_t)rows[j] * cpr + c0 + 64 * u] : zero_chunk();
#pragma unroll
      for (int u = 0; u < CPL; ++u) {
        const int c = c0 + 64 * u;
        float g[N], o[N], sc[N];
        chunk_to_f<T>(gc[u], g);
#pragma unroll
        for (int j = 0; j < KM; ++j) {
          if (rows[j] >= 0 && c < cpr) {
            chunk_to_f<T>(in[j][u], o);
#pragma unroll
            for (int i = 0; i < N; ++i) {
              dot[j] = fmaf(g[i], o[i], dot[j]);
              sc[i] = w[j] * g[i];
            }
            dyp[(size_t)rows[j] * cpr + c] = f_to_chunk<T>(sc);
          }
        }
      }
    }
#pragma unroll
    for (int j = 0; j < KM; ++j) {
      if (j < k) {
        float tot = wave_sum(dot[j]);
        if (lane == 0) dgate[(size_t)t * k + j] = (rows[j] >= 0) ? tot : 0.f;
      }
    }
  }
}

hipError_t launch_combine(const moe_desc& d, const void* yp, const int32_t* s2r, const float* w, void* y,
                          hipStream_t s) {
  const int cpr = (int)(d.d_model * elem_bytes(d) / 16);
  KernelTimer kt("combine", s);
  batch_dispatch(d.top_k, d.n_shared, false, [&](auto km, auto sm, auto) {
    constexpr int KM = decltype(km)::value, SM = decltype(sm)::value;
    if (d.dtype == MOE_BF16)
      hipLaunchKernelGGL((combine_kernel<bf16, KM, SM>), dim3(token_blocks(d.T)), dim3(256), 0, s, d.T, d.top_k,
                         d.n_shared, cpr, (const Chunk*)yp, s2r, w, (Chunk*)y);
    else
      hipLaunchKernelGGL((combine_kernel<float, KM, SM>), dim3(token_blocks(d.T)), dim3(256), 0, s, d.T, d.top_k,
                         d.n_shared, cpr, (const Chunk*)yp, s2r, w, (Chunk*)y);
  });
  return hipGetLastError();
}

hipError_t launch_combine_bwd(const moe_desc& d, const void* dy, const void* yp, const int32_t* s2r,
                              const float* w, void* dyp, float* dgate, hipStream_t s) {
  const int cpr = (int)(d.d_model * elem_bytes(d) / 16);
  KernelTimer kt("combine_bwd", s);
  row_dispatch(d.top_k, cpr, [&](auto km, auto cpl) {
    constexpr int KM = decltype(km)::value, CPL = decltype(cpl)::value;
    if (d.dtype == MOE_BF16)
      hipLaunchKernelGGL((combine_bwd_kernel<bf16, KM, CPL>), dim3(token_blocks(d.T)), dim3(256), 0, s, d.T,
                         d.top_k, cpr, (const Chunk*)dy, (const Chunk*)yp, s2r, w, (Chunk*)dyp, dgate);
    else
      hipLaunchKernelGGL((combine_bwd_kernel<float, KM, CPL>), dim3(token_blocks(d.T)), dim3(256), 0, s, d.T,
                         d.top_k, cpr, (const Chunk*)dy, (const Chunk*)yp, s2r, w, (Chunk*)dyp, dgate);
  });
  return hipGetLastError();
}

}  // namespace pcmoe
