// Grouped-GEMM pieces shared by the bf16 (MFMA 16x16x32, direct-to-LDS) and fp32 kernels.
#pragma once
#include "pcmoe_internal.h"

namespace pcmoe {

enum GemmKind { FWD_GU = 0, FWD_DOWN = 1, BWD_DH = 2, BWD_DX = 3, WG_DOWN = 4, WG_GU = 5 };

struct GemmArgs {
  int T, k, d, f, Eloc, S;
  int rows_cap;               // T*k: first row of the shared experts in the row space
  const int32_t* offsets;     // [Eloc+1]
  const int32_t* mt_prefix;   // [G+1] m-tile prefix of the row-ragged kinds
  const int32_t* order;       // [G] groups by decreasing row count (weight-gradient kinds), or null
  int n_tiles, m_tiles;       // tiles along N (all kinds) and along M (weight-gradient kinds)
  const void* x;              // [T, d]
  const void* xp;             // [T*k, d]
  const void* dy;             // [T, d]
  const void* dyp;            // [T*k, d]
  const void* wg;             // [G, f, d]
  const void* wu;             // [G, f, d]
  const void* wd;             // [G, d, f]
  void* gu;                   // [R, 2f] saved G|U (FWD_GU writes, BWD_DH reads)
  void* h;                    // [R, f] saved H
  void* dgu;                  // [R, 2f] dG|dU
  void* out;                  // y_perm / dx_perm / dW_down / dW_gate
  void* out2;                 // dW_up (WG_GU)
};

template <int KIND> struct KindTraits;
template <> struct KindTraits<FWD_GU> { static constexpr bool ragged_m = true, a_kc = true, b_kc = true; };
template <> struct KindTraits<FWD_DOWN> { static constexpr bool ragged_m = true, a_kc = true, b_kc = true; };
template <> struct KindTraits<BWD_DH> { static constexpr bool ragged_m = true, a_kc = true, b_kc = false; };
template <> struct KindTraits<BWD_DX> { static constexpr bool ragged_m = true, a_kc = true, b_kc = false; };
template <> struct KindTraits<WG_DOWN> { static constexpr bool ragged_m = false, a_kc = false, b_kc = false; };
template <> struct KindTraits<WG_GU> { static constexpr bool ragged_m = false, a_kc = false, b_kc = false; };

constexpr int GROUP_M = 8;  // m-tiles visited together for L2 reuse of the weight tiles

__device__ __forceinline__ int find_group(const int32_t* __restrict__ pre, int G, int L, int nt) {
  int lo = 0, hi = G - 1;  // largest g with pre[g]*nt <= L
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (pre[mid] * nt <= L) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

// Decode a workgroup's tile: XCD-aware order (consecutive logical tiles on one XCD), groups by
// device-side prefix, m-tiles in bunches of GROUP_M per n-tile. Returns false for idle workgroups.
struct TileIdx {
  int g, mt, nt;
};
template <bool RAGGED>
__device__ __forceinline__ bool decode_tile(const GemmArgs& p, int bid, TileIdx& t) {
  const int G = p.Eloc + p.S;
  int total;
  if (RAGGED) total = p.mt_prefix[G] * p.n_tiles;
  else total = G * p.m_tiles * p.n_tiles;
  // Ragged kinds: equal-cost tiles, so each XCD takes a contiguous run of them (its L2 then holds the
  // weights of few groups). Weight-gradient tiles cost K = rows of their group, heaviest groups
  // first; they are dealt round-robin over the XCDs so that the long ones spread out.
  int L;
  if (RAGGED) {
    const int per_xcd = (total + 7) >> 3;
    if ((bid >> 3) >= per_xcd) return false;
    L = (bid & 7) * per_xcd + (bid >> 3);
  } else {
    L = bid;
  }
  if (L >= total) return false;
  int l, n_mt;
  if (RAGGED) {
    t.g = find_group(p.mt_prefix, G, L, p.n_tiles);
    l = L - p.mt_prefix[t.g] * p.n_tiles;
    n_mt = p.mt_prefix[t.g + 1] - p.mt_prefix[t.g];
  } else {
    const int rank = L / (p.m_tiles * p.n_tiles);  // heaviest groups first: their long K loops start early
    t.g = p.order ? p.order[rank] : rank;
    l = L - rank * p.m_tiles * p.n_tiles;
    n_mt = p.m_tiles;
  }
  const int mblk = l / (GROUP_M * p.n_tiles);
  const int rem = l - mblk * GROUP_M * p.n_tiles;
  const int gsz = min(GROUP_M, n_mt - mblk * GROUP_M);
  t.nt = rem / gsz;
  t.mt = mblk * GROUP_M + rem % gsz;
  return true;
}

__global__ __launch_bounds__(512) void mtile_prefix_kernel(const int32_t* __restrict__ offsets, int Eloc, int S,
                                                           int Tn, int bm0, int bm1, int32_t* __restrict__ pre0,
                                                           int32_t* __restrict__ pre1, int32_t* __restrict__ order);

// fp32 path (generic LDS-tiled MFMA 16x16x4 kernel)
hipError_t ffn_fwd_f32(const moe_desc& d, const void* x, const void* xp, const int32_t* offsets, const void* wg,
                       const void* wu, const void* wd, void* yp, void* saved, int32_t* pre, hipStream_t s);
hipError_t ffn_bwd_f32(const moe_desc& d, const void* x, const void* xp, const void* dy, const void* dyp,
                       const int32_t* offsets, const void* wg, const void* wu, const void* wd, const void* saved,
                       void* dxp, void* dwg, void* dwu, void* dwd, void* dgu, int32_t* pre, hipStream_t s);

}  // namespace pcmoe
