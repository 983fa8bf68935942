// Gating (Alg. 7: scores, softmax, TopKIndices, w = p[I]) and its adjoint on the data owner.
//
// Scores are accumulated in fp64 (MFMA f64) from the exact products of the stored inputs and rounded
// once to fp32, so the top-k decision is reproducible from the inputs alone. Selection happens at
// wavefront level: k rounds of a 64-lane butterfly argmax on (score, -expert index).
#include "pcmoe_internal.h"
#include <math.h>

namespace pcmoe {

typedef double doublex4 __attribute__((ext_vector_type(4)));

constexpr int RT_TOK = 16;  // tokens per workgroup (one MFMA row block)

// Scores of 16 tokens against all E experts on v_mfma_f64_16x16x4f64. The W wavefronts split d into
// W equal ranges; their fp64 partial sums are added in a fixed order, the bias is added in fp64 and the
// result is rounded once to fp32. Each lane feeds one 16-byte chunk of its token row and of its
// expert row (8 bf16 / 4 fp32 consecutive k) into 8 / 4 MFMAs: MFMA s takes element s of every
// lane, so lane group q contributes k = 4*EPC*c + EPC*q + s (the same mapping on both operands).
// NET = 16-expert tiles per wavefront (E <= 16 * NET). Each wavefront then selects for 16 / W tokens.
template <typename T, int NET, int W>
__global__ __launch_bounds__(64 * W) void route_fwd_kernel(const T* __restrict__ x, const T* __restrict__ wr,
                                                        const float* __restrict__ bias, int bias_div, int Tn,
                                                        int d, int E, int k, int renorm,
                                                        float* __restrict__ logits, int32_t* __restrict__ idx,
                                                        float* __restrict__ gw) {
  constexpr int EP = EPC<T>::value;   // elements per 16-byte chunk
  constexpr int EW = 16 * NET + 1;    // padded expert stride of the partial-sum table
  extern __shared__ double part[];    // [W waves][16 tokens][EW]
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int i = lane & 15, q = lane >> 4;
  const int t0 = blockIdx.x * RT_TOK;
  const int t = t0 + i;
  const int kq = d / W;
  const int kb = wave * kq;
  // CH independent accumulator chains per expert tile (column steps alternate between them), added in
  // chain order at the end: back-to-back MFMAs on one accumulator wait for each other.
  constexpr int CH = NET <= 4 ? 2 : 1;
  doublex4 acc[CH][NET];
#pragma unroll
  for (int ch = 0; ch < CH; ++ch)
#pragma unroll
    for (int et = 0; et < NET; ++et) acc[ch][et] = doublex4{0.0, 0.0, 0.0, 0.0};
  const T* xrow = x + (size_t)(t < Tn ? t : 0) * d;
  // Column steps of 4 chunks; the loads of the next two steps are in flight while one step computes.
  const int nstep = kq / (4 * EP);
  auto load = [&](int st, Chunk& xc, Chunk (&wc)[NET]) {
    const int c = kb + st * 4 * EP + EP * q;
    xc = t < Tn ? ld_chunk(xrow + c) : zero_chunk();
#pragma unroll
    for (int et = 0; et < NET; ++et) {
      const int e = 16 * et + i;
      wc[et] = e < E ? ld_chunk(wr + (size_t)e * d + c) : zero_chunk();
    }
  };
  auto compute = [&](const Chunk& xc, const Chunk (&wc)[NET]) {
    float xf[EP];
    chunk_to_f<T>(xc, xf);
#pragma unroll
    for (int et = 0; et < NET; ++et) {
      float wf[EP];
      chunk_to_f<T>(wc[et], wf);
#pragma unroll
      for (int s = 0; s < EP; ++s)
        acc[s % CH][et] =
            __builtin_amdgcn_mfma_f64_16x16x4f64((double)xf[s], (double)wf[s], acc[s % CH][et], 0, 0, 0);
    }
  };
  Chunk xa, xb, wa[NET], wb[NET];
  if (nstep > 0) load(0, xa, wa);
  if (nstep > 1) load(1, xb, wb);
  for (int st = 0; st < nstep; st += 2) {
    compute(xa, wa);
    if (st + 2 < nstep) load(st + 2, xa, wa);
    if (st + 1 < nstep) {
      compute(xb, wb);
      if (st + 3 < nstep) load(st + 3, xb, wb);
    }
  }
  // f64 16x16x4 output: register r of lane group q holds D[token 4r + q][expert 16 et + i]
#pragma unroll
  for (int et = 0; et < NET; ++et)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      double a = acc[0][et][r];
#pragma unroll
      for (int ch = 1; ch < CH; ++ch) a += acc[ch][et][r];
      part[(wave * 16 + 4 * r + q) * EW + 16 * et + i] = a;
    }
  __syncthreads();

  // TW tokens per wavefront: fixed-order sum of the W partials, bias, one rounding, then top-k. The
  // tokens of a wavefront go through the cross-lane argmax rounds together, so their shuffle latencies
  // overlap.
  constexpr int TW = RT_TOK / W;  // tokens per wavefront
  float v[TW][4];
  bool taken[TW][4];
#pragma unroll
  for (int rr = 0; rr < TW; ++rr) {
    const int row = wave * TW + rr;
    const int tt = t0 + row;
#pragma unroll
    for (int qq = 0; qq < 4; ++qq) {
      const int e = lane + 64 * qq;
      v[rr][qq] = -INFINITY;
      taken[rr][qq] = true;
      if (tt < Tn && e < E) {
        double sum = part[row * EW + e];
#pragma unroll
        for (int w = 1; w < W; ++w) sum += part[(w * 16 + row) * EW + e];
        if (bias) sum += (double)bias[(size_t)(tt / bias_div) * E + e];
        const float L = (float)sum;
        logits[(size_t)tt * E + e] = L;
        v[rr][qq] = L;
        taken[rr][qq] = false;
      }
    }
  }
  float myv[TW], bv[TW];
  int myi[TW], bi[TW];
#pragma unroll
  for (int rr = 0; rr < TW; ++rr) {
    myv[rr] = -INFINITY;
    myi[rr] = 0;
  }
  for (int j = 0; j < k; ++j) {
#pragma unroll
    for (int rr = 0; rr < TW; ++rr) {
      bv[rr] = -INFINITY;
      bi[rr] = 0x7fffffff;
#pragma unroll
      for (int qq = 0; qq < 4; ++qq) {
        const int e = lane + 64 * qq;
        if (!taken[rr][qq] && (v[rr][qq] > bv[rr] || (v[rr][qq] == bv[rr] && e < bi[rr]))) {
          bv[rr] = v[rr][qq];
          bi[rr] = e;
        }
      }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      float ov[TW];
      int oi[TW];
#pragma unroll
      for (int rr = 0; rr < TW; ++rr) {
        ov[rr] = __shfl_xor(bv[rr], off, 64);
        oi[rr] = __shfl_xor(bi[rr], off, 64);
      }
#pragma unroll
      for (int rr = 0; rr < TW; ++rr)
        if (ov[rr] > bv[rr] || (ov[rr] == bv[rr] && oi[rr] < bi[rr])) {
          bv[rr] = ov[rr];
          bi[rr] = oi[rr];
        }
    }
#pragma unroll
    for (int rr = 0; rr < TW; ++rr) {
#pragma unroll
      for (int qq = 0; qq < 4; ++qq)
        if (lane + 64 * qq == bi[rr]) taken[rr][qq] = true;
      if (lane == j) {
        myv[rr] = bv[rr];
        myi[rr] = bi[rr];
      }
    }
  }
  float ex[TW], zp[TW];
#pragma unroll
  for (int rr = 0; rr < TW; ++rr) {
    const float m = __shfl(myv[rr], 0, 64);  // the largest score of the token
    ex[rr] = (lane < k) ? expf(myv[rr] - m) : 0.f;
    if (renorm) {
      zp[rr] = ex[rr];
    } else {
      zp[rr] = 0.f;
#pragma unroll
      for (int qq = 0; qq < 4; ++qq)
        if (lane + 64 * qq < E) zp[rr] += expf(v[rr][qq] - m);
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1)
#pragma unroll
    for (int rr = 0; rr < TW; ++rr) zp[rr] += __shfl_xor(zp[rr], off, 64);
#pragma unroll
  for (int rr = 0; rr < TW; ++rr) {
    const int tt = t0 + wave * TW + rr;
    if (tt < Tn && lane < k) {
      idx[(size_t)tt * k + lane] = myi[rr];
      gw[(size_t)tt * k + lane] = ex[rr] / zp[rr];
    }
  }
}

template <typename T>
static hipError_t route_fwd_t(const moe_desc& d, const void* x, const void* wr, const float* bias, int bg,
                              float* logits, int32_t* idx, float* w, hipStream_t s) {
  const int E = d.n_experts;
  dim3 grid((d.T + RT_TOK - 1) / RT_TOK);
  const int div = d.T / (bg > 0 ? bg : 1);
  KernelTimer kt("route_fwd", s);
  // Wavefronts per workgroup: as many as split d into whole column steps (4 chunks) and keep the
  // partial-sum table within 64 KB (all 4 beyond that: d is a multiple of 128).
  constexpr int STEP = 4 * EPC<T>::value;
  auto waves_for = [&](int net) {
    for (int wv = 16; wv > 4; wv >>= 1)
      if (d.d_model % (wv * STEP) == 0 && (size_t)wv * 16 * (16 * net + 1) * sizeof(double) <= 65536) return wv;
    return 4;
  };
#define RT_LAUNCH_W(NET, W)                                                                                     \
  do {                                                                                                          \
    const size_t lds = (size_t)W * 16 * (16 * NET + 1) * sizeof(double);                                       \
    if (lds > 65536) {                                                                                          \
      static std::atomic<uint64_t> lds_set_{0};                                                                 \
      hipError_t e_ = lds_limit_once((const void*)route_fwd_kernel<T, NET, W>, (int)lds, lds_set_);             \
      if (e_ != hipSuccess) return e_;                                                                          \
    }                                                                                                           \
    hipLaunchKernelGGL((route_fwd_kernel<T, NET, W>), grid, dim3(64 * W), lds, s, (const T*)x, (const T*)wr,     \
                       bias, div, d.T, d.d_model, E, d.top_k, d.renormalize, logits, idx, w);                   \
  } while (0)
  // (the table limit leaves 16 wavefronts to NET = 1 and 8 to NET <= 2)
  if (E <= 16) {
    const int wv = waves_for(1);
    if (wv == 16) RT_LAUNCH_W(1, 16);
    else if (wv == 8) RT_LAUNCH_W(1, 8);
    else RT_LAUNCH_W(1, 4);
  } else if (E <= 32) {
    if (waves_for(2) == 8) RT_LAUNCH_W(2, 8);
    else RT_LAUNCH_W(2, 4);
  } else if (E <= 64) {
    RT_LAUNCH_W(4, 4);
  } else if (E <= 128) {
    RT_LAUNCH_W(8, 4);
  } else {
    RT_LAUNCH_W(16, 4);
  }
#undef RT_LAUNCH_W
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

// Partial dW_router over one chunk of tokens, part[chunk][e][c] = sum_{t in chunk} dl[t][e] * x[t][c], as an
// fp32 MFMA contraction (v_mfma_f32_16x16x4f32, tokens as K). Lane (q, i) of a wavefront loads JJ contiguous
// columns c0 + JJ*i .. + JJ-1 of token rows t + q (one coalesced load of the row segment per 16 lanes) and
// feeds column c0 + JJ*i + jj of MFMA number jj; its A operand is dl[t + q][16 et + i]. 8 token-steps of 4
// tokens are loaded before their MFMAs.
template <typename T, int JJ>
struct alignas(JJ * sizeof(T) < 16 ? JJ * sizeof(T) : 16) XRow {  // tensors are 16-byte aligned
  T v[JJ];
};

// JJ columns per lane: 4 for up to 16 experts (narrower workgroups, so that 256 of them need only 64 token
// chunks of partial sums: measured 9 us against 12 us for 8 columns and 128 chunks at T=4096, d=1024), 8 while the
// accumulators (JJ x NET tiles) fit, fewer for many experts.
constexpr int dw_cols_per_lane(int net) { return net == 1 ? 4 : net <= 2 ? 8 : 16 / net > 0 ? 16 / net : 1; }

template <typename T, int NET, int JJ>
__global__ __launch_bounds__(256) void route_dw_partial_kernel(int Tn, int d, int E, int tok_per_chunk,
                                                               const T* __restrict__ x,
                                                               const float* __restrict__ dl,
                                                               float* __restrict__ part) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int q = lane >> 4, i = lane & 15;
  const int c0 = (blockIdx.x * 4 + wave) * 16 * JJ;  // first column of this wavefront
  if (c0 >= d) return;                               // d is a multiple of 16 * JJ: all or nothing
  const int chunk = blockIdx.y;
  const int tb = chunk * tok_per_chunk;
  const int te = min(Tn, tb + tok_per_chunk);
  floatx4 acc[JJ][NET];
#pragma unroll
  for (int jj = 0; jj < JJ; ++jj)
#pragma unroll
    for (int et = 0; et < NET; ++et) acc[jj][et] = floatx4{0.f, 0.f, 0.f, 0.f};
  for (int t0 = tb; t0 < te; t0 += 32) {
    XRow<T, JJ> xv[8];
    float a[8][NET];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int t = t0 + 4 * u + q;
      const bool ok = t < te;
      if (ok) xv[u] = *reinterpret_cast<const XRow<T, JJ>*>(x + (size_t)t * d + c0 + JJ * i);
      else xv[u] = XRow<T, JJ>{};
#pragma unroll
      for (int et = 0; et < NET; ++et) {
        const int e = 16 * et + i;
        a[u][et] = (ok && e < E) ? dl[(size_t)t * E + e] : 0.f;
      }
    }
#pragma unroll
    for (int u = 0; u < 8; ++u)
#pragma unroll
      for (int jj = 0; jj < JJ; ++jj) {
        const float b = to_f(xv[u].v[jj]);
#pragma unroll
        for (int et = 0; et < NET; ++et)
          acc[jj][et] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[u][et], b, acc[jj][et], 0, 0, 0);
      }
  }
  // register r of lane group q holds D[expert 16 et + 4q + r][n = i], column c0 + JJ*i + jj
#pragma unroll
  for (int et = 0; et < NET; ++et)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int e = 16 * et + 4 * q + r;
      if (e >= E) continue;
      float* o = part + ((size_t)chunk * E + e) * d + c0 + JJ * i;
#pragma unroll
      for (int jj = 0; jj < JJ; ++jj) o[jj] = acc[jj][et][r];
    }
}

// dW_router[o] = sum over chunks of part[chunk][o], in a fixed order: thread (g, o) of a workgroup sums
// the chunks g, g + 16, g + 32, ... in turn, then the 16 partial sums of an output are added in g order.
constexpr int RED_G = 16;  // chunk lanes per output
__global__ __launch_bounds__(256) void route_dw_reduce_kernel(int n4, int nchunks, const float4* __restrict__ part,
                                                              float4* __restrict__ out) {
  __shared__ float4 red[RED_G][256 / RED_G];
  const int g = threadIdx.x / (256 / RED_G), ol = threadIdx.x % (256 / RED_G);
  const int o = blockIdx.x * (256 / RED_G) + ol;
  float4 s = float4{0.f, 0.f, 0.f, 0.f};
  if (o < n4)
    for (int c = g; c < nchunks; c += RED_G) {
      const float4 v = part[(size_t)c * n4 + o];
      s.x += v.x;
      s.y += v.y;
      s.z += v.z;
      s.w += v.w;
    }
  red[g][ol] = s;
  __syncthreads();
  if (g == 0 && o < n4) {
    float4 t = red[0][ol];
    for (int h = 1; h < RED_G; ++h) {
      const float4 v = red[h][ol];
      t.x += v.x;
      t.y += v.y;
      t.z += v.z;
      t.w += v.w;
    }
    out[o] = t;
  }
}

static int dw_net(int E) { return E <= 16 ? 1 : E <= 32 ? 2 : E <= 64 ? 4 : E <= 128 ? 8 : 16; }

// Token chunks of the weight-gradient contraction: enough workgroups to fill the chip, chunk sizes a
// multiple of 32 tokens. A workgroup covers 4 wavefronts x 16 x JJ columns.
// Workgroups of the partial contraction: about 256 for up to 16 experts, 1024 for more.
static void route_bwd_chunks(const moe_desc& d, int* nch, int* tpc) {
  const int net = dw_net(d.n_experts);
  const int wg_cols = 64 * dw_cols_per_lane(net);
  const int ncol = (d.d_model + wg_cols - 1) / wg_cols;
  const int maxch = (d.T + 31) / 32;
  const int target = net == 1 ? 256 : 1024;
  int want = (target + ncol - 1) / ncol;
  int n = want < maxch ? want : maxch;
  if (n < 1) n = 1;
  int per = (d.T + n - 1) / n;
  per = ((per + 31) / 32) * 32;
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
    const int wg_cols = 64 * dw_cols_per_lane(dw_net(E));
    dim3 grid((d.d_model + wg_cols - 1) / wg_cols, nch);
#define RB_LAUNCH(NET)                                                                                           \
  hipLaunchKernelGGL((route_dw_partial_kernel<T, NET, dw_cols_per_lane(NET)>), grid, dim3(256), 0, s, d.T,     \
                     d.d_model, E, tpc, (const T*)x, dl, part)
    if (E <= 16) RB_LAUNCH(1);
    else if (E <= 32) RB_LAUNCH(2);
    else if (E <= 64) RB_LAUNCH(4);
    else if (E <= 128) RB_LAUNCH(8);
    else RB_LAUNCH(16);
#undef RB_LAUNCH
  }
  {
    KernelTimer kt("route_dw_reduce", s);
    const int n4 = E * d.d_model / 4;
    const int blocks = (n4 + 256 / RED_G - 1) / (256 / RED_G);
    hipLaunchKernelGGL(route_dw_reduce_kernel, dim3(blocks), dim3(256), 0, s, n4, nch, (const float4*)part,
                       (float4*)dwr);
  }
  return hipGetLastError();
}

hipError_t launch_route_bwd(const moe_desc& d, const void* x, const float* logits, const int32_t* idx,
                            const float* w, const float* dgate, float* dl, float* dwr, void* ws, hipStream_t s) {
  if (d.dtype == MOE_BF16) return route_bwd_t<bf16>(d, x, logits, idx, w, dgate, dl, dwr, ws, s);
  return route_bwd_t<float>(d, x, logits, idx, w, dgate, dl, dwr, ws, s);
}

}  // namespace pcmoe
