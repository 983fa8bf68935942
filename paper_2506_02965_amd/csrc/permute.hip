// Dispatch of Alg. 3 (each token's hidden state goes to the host of every expert it selected) as a stable counting sort
// of the hosted assignment slots a = t*k + j by expert, plus the gather of their token rows;
// and the hand-back of the input gradient (Sec. 3.2), summed per token.
//
// Ordering is reproducible bit for bit: rows of one expert are in increasing slot order.
//   1. histogram: per block of PM_SLOTS slots, per hosted expert counts (LDS atomics; order-free)
//   2. scatter: each block first derives its own base per expert from the histogram (the exclusive
//      prefix over experts of the totals, plus the counts of the earlier blocks; block 0 also writes
//      counts and offsets), then each wavefront ranks its 64 slots with ballots (lanes holding the
//      same expert form a peer mask; rank = popcount of lower peers), waves in order.
//   3. gather: one wavefront per token reads its row once and writes its k destinations.
#include "pcmoe_internal.h"

namespace pcmoe {

constexpr int PM_SLOTS = 1024;  // slots per block (4 waves x 4 x 64)

__device__ __forceinline__ uint64_t peer_mask(int v, bool valid, int nbits) {
  uint64_t peers = __ballot(valid);
  for (int b = 0; b < nbits; ++b) {
    const bool bit = (v >> b) & 1;
    const uint64_t m = __ballot(bit);
    peers &= bit ? m : ~m;
  }
  return peers;
}

__global__ __launch_bounds__(256) void perm_hist_kernel(const int32_t* __restrict__ idx, int nslots, int lb,
                                                        int lc, int32_t* __restrict__ blk_counts) {
  extern __shared__ int hist[];
  for (int e = threadIdx.x; e < lc; e += 256) hist[e] = 0;
  __syncthreads();
  const int a0 = blockIdx.x * PM_SLOTS;
  for (int i = threadIdx.x; i < PM_SLOTS; i += 256) {
    int a = a0 + i;
    if (a < nslots) {
      int v = idx[a] - lb;
      if (v >= 0 && v < lc) atomicAdd(&hist[v], 1);
    }
  }
  __syncthreads();
  for (int e = threadIdx.x; e < lc; e += 256) blk_counts[(size_t)blockIdx.x * lc + e] = hist[e];
}

__global__ __launch_bounds__(256) void perm_scatter_kernel(const int32_t* __restrict__ idx, int nslots, int lb,
                                                           int lc, int nbits, int nblk,
                                                           const int32_t* __restrict__ blk_counts,
                                                           int32_t* __restrict__ counts, int32_t* __restrict__ offsets,
                                                           int32_t* __restrict__ r2s, int32_t* __restrict__ s2r) {
  extern __shared__ int wcnt[];  // [4][lc]
  __shared__ int base[256];      // this block's first row per expert
  __shared__ int wsum[4];
  __shared__ int nloc_s;
  __shared__ int part_before[256], part_tot[256];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  constexpr int ITERS = PM_SLOTS / 4 / 64;  // slots of a lane: a wave ranks its PM_SLOTS / 4 slots 64 at a time
  const int a_w = blockIdx.x * PM_SLOTS + w * (PM_SLOTS / 4);
  // the local expert of each of the lane's slots (-1: hosted elsewhere or past the end), loaded once, in flight
  // together with the count-table loads below
  int v_of[ITERS];
#pragma unroll
  for (int it = 0; it < ITERS; ++it) {
    const int a = a_w + it * 64 + lane;
    const int v = (a < nslots) ? idx[a] - lb : -1;
    v_of[it] = (v >= 0 && v < lc) ? v : -1;
  }
  for (int i = threadIdx.x; i < 4 * lc; i += 256) wcnt[i] = 0;
  {
    // Per expert, the rows of the earlier blocks and the total over all blocks. The nblk x lc count table is
    // split over the block's threads: lcp (lc rounded up to a power of two, <= 256) experts by 256 / lcp parts
    // of the blocks, each thread summing its part's column with its loads in flight together; the parts are
    // then added in LDS, in part order.
    const int lcp = lc <= 1 ? 1 : 1 << (32 - __builtin_clz(lc - 1));
    const int nparts = 256 / lcp;
    const int ep = threadIdx.x & (lcp - 1), part = threadIdx.x / lcp;
    const int chunk = (nblk + nparts - 1) / nparts;
    const int b0 = part * chunk, b1 = min(nblk, b0 + chunk);
    int pb = 0, pt = 0;
    if (ep < lc) {
#pragma unroll 8
      for (int b = b0; b < b1; ++b) {
        const int c = blk_counts[(size_t)b * lc + ep];
        pb += (b < (int)blockIdx.x) ? c : 0;
        pt += c;
      }
    }
    part_before[threadIdx.x] = pb;
    part_tot[threadIdx.x] = pt;
    __syncthreads();
    // expert e = thread: then the exclusive prefix of the totals over experts (lc <= 256)
    const int e = threadIdx.x;
    int tot = 0, before = 0;
    if (e < lc)
      for (int q = 0; q < nparts; ++q) {
        before += part_before[q * lcp + e];
        tot += part_tot[q * lcp + e];
      }
    int incl = tot;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int o = __shfl_up(incl, off, 64);
      if (lane >= off) incl += o;
    }
    if (lane == 63) wsum[w] = incl;
    __syncthreads();
    int wb = 0;
    for (int i = 0; i < w; ++i) wb += wsum[i];
    const int excl = wb + incl - tot;
    base[e] = excl + before;
    if (e == 255) nloc_s = wb + incl;  // rows of all hosted experts
    if (blockIdx.x == 0 && e < lc) {
      counts[e] = tot;
      offsets[e] = excl;
      if (e == lc - 1) offsets[lc] = excl + tot;
    }
  }
  __syncthreads();
  const uint64_t lt = (lane == 0) ? 0ull : ((~0ull) >> (64 - lane));
  int* mine = wcnt + w * lc;
  // pass 1: per-wave counts
#pragma unroll
  for (int it = 0; it < ITERS; ++it) {
    const int v = v_of[it];
    const uint64_t peers = peer_mask(v < 0 ? 0 : v, v >= 0, nbits);
    if (v >= 0 && (peers & lt) == 0) mine[v] += __popcll(peers);
  }
  __syncthreads();
  for (int e = threadIdx.x; e < lc; e += 256) {
    int r = base[e];
    for (int ww = 0; ww < 4; ++ww) {
      int c = wcnt[ww * lc + e];
      wcnt[ww * lc + e] = r;
      r += c;
    }
  }
  __syncthreads();
  // pass 2: stable ranks
#pragma unroll
  for (int it = 0; it < ITERS; ++it) {
    const int a = a_w + it * 64 + lane;
    const int v = v_of[it];
    const uint64_t peers = peer_mask(v < 0 ? 0 : v, v >= 0, nbits);
    if (a < nslots) {
      if (v >= 0) {
        const int pos = mine[v] + __popcll(peers & lt);
        r2s[pos] = a;
        s2r[a] = pos;
      } else {
        s2r[a] = -1;
      }
    }
    if (v >= 0 && (peers & lt) == 0) mine[v] += __popcll(peers);
  }
  // rows beyond N_loc have no slot
  const int nloc = nloc_s;
  for (int i = threadIdx.x; i < PM_SLOTS; i += 256) {
    int r = blockIdx.x * PM_SLOTS + i;
    if (r < nslots && r >= nloc) r2s[r] = -1;
  }
}

// Token-major gather: x_perm[slot_to_row[t*k+j]] = x[t] for every hosted slot.
// One wavefront per token. Each lane handles CPL 16-byte chunks of the row per pass, loaded together, so a
// token costs one round trip for its slot map and its row, not one per chunk.
template <int KM, int CPL>
__global__ __launch_bounds__(256) void perm_gather_kernel(int Tn, int k, int cpr, const Chunk* __restrict__ x,
                                                          const int32_t* __restrict__ s2r, Chunk* __restrict__ xp) {
  const int lane = threadIdx.x & 63;
  const int wave = (blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int nwaves = (gridDim.x * blockDim.x) >> 6;
  for (int t = wave; t < Tn; t += nwaves) {
    int rows[KM];
#pragma unroll
    for (int j = 0; j < KM; ++j) rows[j] = (j < k) ? s2r[(size_t)t * k + j] : -1;
    for (int c0 = lane; c0 < cpr; c0 += 64 * CPL) {
      Chunk v[CPL];
#pragma unroll
      for (int u = 0; u < CPL; ++u) v[u] = (c0 + 64 * u < cpr) ? x[(size_t)t * cpr + c0 + 64 * u] : zero_chunk();
#pragma unroll
      for (int u = 0; u < CPL; ++u) {
        const int c = c0 + 64 * u;
        if (c < cpr) {
#pragma unroll
          for (int j = 0; j < KM; ++j)
            if (rows[j] >= 0) xp[(size_t)rows[j] * cpr + c] = v[u];
        }
      }
    }
  }
}

static int nbits_for(int lc) {
  int nb = 0;
  while ((1 << nb) < lc) ++nb;
  return nb;
}

size_t permute_ws_bytes(const moe_desc& d) {
  size_t nslots = (size_t)d.T * d.top_k;
  size_t nblk = (nslots + PM_SLOTS - 1) / PM_SLOTS;
  return align256(nblk * d.local_count * sizeof(int32_t));
}

// ------------------------------------------------------------------ allocation-free dispatch
// The scratch of moe_permute_noalloc: the per-block expert counts (ceil(T*k / PM_SLOTS) x local_count int32) in a
// device array of fixed size. Each GPU the library runs on holds its own copy until the process ends; every call
// on that GPU shares it. Nothing in it needs clearing: the histogram launch writes every count the scatter reads.
constexpr size_t kNoallocScratchBytes = size_t(1) << 20;
static __device__ __align__(256) char scratch[kNoallocScratchBytes];

size_t permute_noalloc_capacity() { return kNoallocScratchBytes; }

// Device address of `scratch` on the current device, looked up once per device with that device current.
// The array's host-side name is no device address: kernels and copies take the pointer returned here.
hipError_t permute_noalloc_scratch(void** out) {
  static std::atomic<void*> addr[64];
  int dev = 0;
  if (hipError_t e = hipGetDevice(&dev); e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  void* p = addr[dev].load(std::memory_order_acquire);
  if (!p) {
    if (hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)); e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    addr[dev].store(p, std::memory_order_release);  // concurrent first calls store the same address
  }
  *out = p;
  return hipSuccess;
}

static int gather_blocks(int Tn) {
  int b = (Tn + 3) / 4;
  return b > 8192 ? 8192 : (b < 1 ? 1 : b);
}

hipError_t launch_permute(const moe_desc& d, const int32_t* idx, const void* x, int32_t* counts, int32_t* offsets,
                          int32_t* r2s, int32_t* s2r, void* xp, void* ws, hipStream_t s) {
  const int nslots = d.T * d.top_k;
  const int nblk = (nslots + PM_SLOTS - 1) / PM_SLOTS;
  const int lc = d.local_count;
  int32_t* blk_counts = (int32_t*)ws;
  {
    KernelTimer kt("permute_hist", s);
    hipLaunchKernelGGL(perm_hist_kernel, dim3(nblk), dim3(256), lc * sizeof(int), s, idx, nslots, d.local_begin, lc,
                       blk_counts);
  }
  {
    KernelTimer kt("permute_scatter", s);
    hipLaunchKernelGGL(perm_scatter_kernel, dim3(nblk), dim3(256), 4 * lc * sizeof(int), s, idx, nslots,
                       d.local_begin, lc, nbits_for(lc), nblk, blk_counts, counts, offsets, r2s, s2r);
  }
  {
    KernelTimer kt("permute_gather", s);
    const int cpr = (int)(d.d_model * elem_bytes(d) / 16);
    row_dispatch(d.top_k, cpr, [&](auto km, auto cpl) {
      hipLaunchKernelGGL((perm_gather_kernel<decltype(km)::value, decltype(cpl)::value>), dim3(gather_blocks(d.T)),
                         dim3(256), 0, s, d.T, d.top_k, cpr, (const Chunk*)x, s2r, (Chunk*)xp);
    });
  }
  return hipGetLastError();
}

// dx_t = sum_j dx_perm[row(t,j)] + sum_s dx_perm[T*k + s*T + t] (+ sum_e dlogits[t,e] * w_router[e])
// One wavefront per token. The token's dlogits row is read once, together with its slot map; its nonzero
// experts (k of them when the gate weights are renormalised) are found with ballots. Each pass loads, in one
// round trip, CPL chunks per lane of the token's KM routed rows, of up to SM shared-expert rows and of the router
// rows of its first RB nonzero experts; further shared experts and nonzero experts follow in later round trips.
// The sums run in slot order, then shared experts, then experts in increasing index.
template <typename T, int KM, int SM, bool DL>
__global__ __launch_bounds__(256) void unpermute_kernel(int Tn, int k, int S, int E, int cpr,
                                                        const Chunk* __restrict__ dxp,
                                                        const int32_t* __restrict__ s2r,
                                                        const float* __restrict__ dl,
                                                        const Chunk* __restrict__ wr, Chunk* __restrict__ dx) {
  constexpr int N = EPC<T>::value;
  constexpr int RB = DL ? KM : 0;
  constexpr int CPL = chunks_per_lane(KM + SM + RB);
  const int lane = threadIdx.x & 63;
  const int wave = (blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int nwaves = (gridDim.x * blockDim.x) >> 6;
  const size_t shared_base = (size_t)Tn * k;
  for (int t = wave; t < Tn; t += nwaves) {
    int rows[KM];
#pragma unroll
    for (int j = 0; j < KM; ++j) rows[j] = (j < k) ? s2r[(size_t)t * k + j] : -1;
    float g[4] = {0.f, 0.f, 0.f, 0.f};
    uint64_t rem[4] = {0ull, 0ull, 0ull, 0ull};
    if (DL) {
#pragma unroll
      for (int qq = 0; qq < 4; ++qq) {
        const int e = lane + 64 * qq;
        g[qq] = (e < E) ? dl[(size_t)t * E + e] : 0.f;
      }
#pragma unroll
      for (int qq = 0; qq < 4; ++qq) rem[qq] = __ballot(g[qq] != 0.f);
    }
    // the first RB nonzero experts in increasing order (wave-uniform), taken out of rem
    int eb[RB > 0 ? RB : 1];
    float gb[RB > 0 ? RB : 1];
#pragma unroll
    for (int b = 0; b < RB; ++b) {
      eb[b] = -1;
      gb[b] = 0.f;
      const int qs = rem[0] ? 0 : rem[1] ? 1 : rem[2] ? 2 : rem[3] ? 3 : -1;
      if (qs >= 0) {
        const uint64_t m = qs == 0 ? rem[0] : qs == 1 ? rem[1] : qs == 2 ? rem[2] : rem[3];
        const float gq = qs == 0 ? g[0] : qs == 1 ? g[1] : qs == 2 ? g[2] : g[3];
        const int l = __builtin_ctzll(m);
        eb[b] = l + 64 * qs;
        gb[b] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(gq), l));
#pragma unroll
        for (int qq = 0; qq < 4; ++qq)
          if (qq == qs) rem[qq] &= rem[qq] - 1;
      }
    }
    for (int c0 = lane; c0 < cpr; c0 += 64 * CPL) {
      Chunk in[KM][CPL], sh[SM > 0 ? SM : 1][CPL], wb[RB > 0 ? RB : 1][CPL];
#pragma unroll
      for (int j = 0; j < KM; ++j)
#pragma unroll
        for (int u = 0; u < CPL; ++u)
          in[j][u] = (rows[j] >= 0 && c0 + 64 * u < cpr) ? dxp[(size_t)rows[j] * cpr + c0 + 64 * u] : zero_chunk();
#pragma unroll
      for (int s = 0; s < SM; ++s)
#pragma unroll
        for (int u = 0; u < CPL; ++u)
          sh[s][u] = (c0 + 64 * u < cpr) ? dxp[(shared_base + (size_t)s * Tn + t) * cpr + c0 + 64 * u] : zero_chunk();
#pragma unroll
      for (int b = 0; b < RB; ++b)
#pragma unroll
        for (int u = 0; u < CPL; ++u)
          wb[b][u] = (eb[b] >= 0 && c0 + 64 * u < cpr) ? wr[(size_t)eb[b] * cpr + c0 + 64 * u] : zero_chunk();
      float acc[CPL][N], v[N];
#pragma unroll
      for (int u = 0; u < CPL; ++u) {
#pragma unroll
        for (int i = 0; i < N; ++i) acc[u][i] = 0.f;
#pragma unroll
        for (int j = 0; j < KM; ++j) {
          if (rows[j] >= 0) {
            chunk_to_f<T>(in[j][u], v);
#pragma unroll
            for (int i = 0; i < N; ++i) acc[u][i] += v[i];
          }
        }
#pragma unroll
        for (int s = 0; s < SM; ++s) {
          chunk_to_f<T>(sh[s][u], v);
#pragma unroll
          for (int i = 0; i < N; ++i) acc[u][i] += v[i];
        }
      }
      for (int s = SM; s < S; ++s) {
#pragma unroll
        for (int u = 0; u < CPL; ++u) {
          if (c0 + 64 * u < cpr) {
            chunk_to_f<T>(dxp[(shared_base + (size_t)s * Tn + t) * cpr + c0 + 64 * u], v);
#pragma unroll
            for (int i = 0; i < N; ++i) acc[u][i] += v[i];
          }
        }
      }
#pragma unroll
      for (int b = 0; b < RB; ++b) {
        if (eb[b] >= 0) {
#pragma unroll
          for (int u = 0; u < CPL; ++u) {
            chunk_to_f<T>(wb[b][u], v);
#pragma unroll
            for (int i = 0; i < N; ++i) acc[u][i] = fmaf(gb[b], v[i], acc[u][i]);
          }
        }
      }
#pragma unroll
      for (int qq = 0; qq < 4; ++qq) {
        uint64_t m = rem[qq];
        while (m) {  // wave-uniform: the remaining nonzero experts, up to four per round, in increasing order
          int es[4];
          float ge[4];
#pragma unroll
          for (int b = 0; b < 4; ++b) {
            es[b] = -1;
            ge[b] = 0.f;
            if (m) {
              const int l = __builtin_ctzll(m);
              m &= m - 1;
              es[b] = l + 64 * qq;
              ge[b] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(g[qq]), l));
            }
          }
          Chunk wv[4][CPL];
#pragma unroll
          for (int b = 0; b < 4; ++b)
#pragma unroll
            for (int u = 0; u < CPL; ++u)
              wv[b][u] = (es[b] >= 0 && c0 + 64 * u < cpr) ? wr[(size_t)es[b] * cpr + c0 + 64 * u] : zero_chunk();
#pragma unroll
          for (int b = 0; b < 4; ++b) {
            if (es[b] >= 0) {
#pragma unroll
              for (int u = 0; u < CPL; ++u) {
                chunk_to_f<T>(wv[b][u], v);
#pragma unroll
                for (int i = 0; i < N; ++i) acc[u][i] = fmaf(ge[b], v[i], acc[u][i]);
              }
            }
          }
        }
      }
#pragma unroll
      for (int u = 0; u < CPL; ++u)
        if (c0 + 64 * u < cpr) dx[(size_t)t * cpr + c0 + 64 * u] = f_to_chunk<T>(acc[u]);
    }
  }
}

hipError_t launch_permute_bwd(const moe_desc& d, const void* dxp, const int32_t* s2r, const float* dl,
                              const void* wr, void* dx, hipStream_t s) {
  const int cpr = (int)(d.d_model * elem_bytes(d) / 16);
  KernelTimer kt("unpermute", s);
  batch_dispatch(d.top_k, d.n_shared, dl != nullptr, [&](auto km, auto sm, auto has_dl) {
    constexpr int KM = decltype(km)::value, SM = decltype(sm)::value;
    constexpr bool DL = decltype(has_dl)::value;
    if (d.dtype == MOE_BF16)
      hipLaunchKernelGGL((unpermute_kernel<bf16, KM, SM, DL>), dim3(gather_blocks(d.T)), dim3(256), 0, s, d.T,
                         d.top_k, d.n_shared, d.n_experts, cpr, (const Chunk*)dxp, s2r, dl, (const Chunk*)wr,
                         (Chunk*)dx);
    else
      hipLaunchKernelGGL((unpermute_kernel<float, KM, SM, DL>), dim3(gather_blocks(d.T)), dim3(256), 0, s, d.T,
                         d.top_k, d.n_shared, d.n_experts, cpr, (const Chunk*)dxp, s2r, dl, (const Chunk*)wr,
                         (Chunk*)dx);
  });
  return hipGetLastError();
}

}  // namespace pcmoe
