// Grouped-GEMM pieces shared by the bf16 (MFMA 16x16x32, direct-to-LDS) and fp32 kernels.
#pragma once
#include "pcmoe_internal.h"

namespace pcmoe {

enum GemmKind { FWD_GU = 0, FWD_DOWN = 1, BWD_DH = 2, BWD_DX = 3, WG_DOWN = 4, WG_GU = 5 };

struct GemmArgs {
  int T, k, d, f, Eloc, S;
  int rows_cap;               // T*k: first row of the shared experts in the row space
  const int32_t* offsets;     // [Eloc+1]
  const int32_t* mt_prefix;   // [G+1] m-tile prefix of the row-ragged kinds (without the tails when mt_tail is set)
  const int32_t* mt_tail;     // [G+1] prefix of the groups' tail m-tiles (at most half their rows), or null
  const int32_t* order;       // [G] groups by decreasing row count (weight-gradient kinds), or null
  int n_tiles, m_tiles;       // tiles along N (all kinds) and along M (weight-gradient kinds)
  int n_extent;               // output columns of the tile grid (FWD_GU: 2f); the last n-tile may hold fewer
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
  int wg_interleave;          // weight gradients: with near-equal groups (order[G] = 1), tile L belongs to group
                              // order[L % G] (round-robin over groups)
  int* tickets;               // single-contraction bf16 launches: a zeroed counter for ticket-claimed tiles, or null
  int tail_split;             // with mt_tail: split each tail tile into up to this many column windows (0 or 1: none)
  int tail_cus;               // ... as long as all the windows fit this many workgroups (the chip's CUs)
};

template <int KIND> struct KindTraits;
template <> struct KindTraits<FWD_GU> { static constexpr bool ragged_m = true, a_kc = true, b_kc = true; };
template <> struct KindTraits<FWD_DOWN> { static constexpr bool ragged_m = true, a_kc = true, b_kc = true; };
template <> struct KindTraits<BWD_DH> { static constexpr bool ragged_m = true, a_kc = true, b_kc = false; };
template <> struct KindTraits<BWD_DX> { static constexpr bool ragged_m = true, a_kc = true, b_kc = false; };
template <> struct KindTraits<WG_DOWN> { static constexpr bool ragged_m = false, a_kc = false, b_kc = false; };
template <> struct KindTraits<WG_GU> { static constexpr bool ragged_m = false, a_kc = false, b_kc = false; };

constexpr int GROUP_M = 8;  // m-tiles visited together for L2 reuse of the weight tiles

// Entry i (wave-uniform) of a small device array spread over the wavefront: lane l holds entry
// 64 * s + l in v[s].
template <int NS>
__device__ __forceinline__ int wave_pick(const int (&v)[NS], int i) {
  int r = 0;
#pragma unroll
  for (int s = 0; s < NS; ++s)
    if ((i >> 6) == s) r = __builtin_amdgcn_readlane(v[s], i & 63);
  return __builtin_amdgcn_readfirstlane(r);  // keeps the result in a scalar register
}

// Decode a workgroup's tile: XCD-aware order (consecutive logical tiles on one XCD), groups by
// device-side prefix, m-tiles in bunches of GROUP_M per n-tile. Returns false for idle workgroups.
// Called by every lane of the wavefront.
struct TileIdx {
  int g, mt, nt;
  int row0, rows;  // the group's first row in its source and its row count
  int sub, nsub;   // column window sub of nsub equal windows: a split tail tile's (nsub = tail_split), else 0 of 1
};
// The plan arrays a tile decode reads, spread over the wavefront (entry 64 s + lane in slot s).
struct DecodeArrays {
  static constexpr int NS = 8;  // 8 x 64 entries per array: groups <= 511
  int pre[NS], ord[NS], off[NS], tl[NS];
};
// One batch of independent loads (a chain of dependent ones costs a memory latency each): the m-tile prefix (ragged
// kinds), the group order (weight gradients) and the row offsets.
template <bool RAGGED>
__device__ __forceinline__ void decode_load(const GemmArgs& p, DecodeArrays& a) {
  const int G = p.Eloc + p.S;
  const int lane = threadIdx.x & 63;
  const int ns = (G + 64) >> 6;  // slots covering entries 0..G
  const bool split = RAGGED && p.mt_tail != nullptr;
#pragma unroll
  for (int s = 0; s < DecodeArrays::NS; ++s) {
    const int i = 64 * s + lane;
    a.pre[s] = 0;
    a.ord[s] = 0;
    a.off[s] = 0;
    a.tl[s] = 0;
    if (s < ns) {
      if (RAGGED && i <= G) a.pre[s] = p.mt_prefix[i];
      if (split && i <= G) a.tl[s] = p.mt_tail[i];
      if (!RAGGED && p.order && i <= G) a.ord[s] = p.order[i];
      if (p.Eloc > 0 && i <= p.Eloc) a.off[s] = p.offsets[i];
    }
  }
}
template <bool RAGGED>
__device__ __forceinline__ bool decode_with(const GemmArgs& p, int bid, const DecodeArrays& a, TileIdx& t);
template <bool RAGGED>
__device__ __forceinline__ bool decode_tile(const GemmArgs& p, int bid, TileIdx& t) {
  DecodeArrays a;
  decode_load<RAGGED>(p, a);
  return decode_with<RAGGED>(p, bid, a, t);
}
// The decode proper, from arrays loaded by decode_load (a persistent workgroup loads them once).
template <bool RAGGED>
__device__ __forceinline__ bool decode_with(const GemmArgs& p, int bid, const DecodeArrays& a, TileIdx& t) {
  constexpr int NS = DecodeArrays::NS;
  const int G = p.Eloc + p.S;
  const int lane = threadIdx.x & 63;
  const int ns = (G + 64) >> 6;
  const bool split = RAGGED && p.mt_tail != nullptr;
  const auto& pre = a.pre;
  const auto& ord = a.ord;
  const auto& off = a.off;
  const auto& tl = a.tl;
  int total;
  if (RAGGED) total = wave_pick(pre, G) * p.n_tiles;
  else total = G * p.m_tiles * p.n_tiles;
  // Ragged kinds: equal-cost tiles, so each XCD takes a contiguous run of them (its L2 then holds the
  // weights of few groups). With mt_tail, a group's last m-tile holding at most half a tile of rows (its
  // empty wavefronts skip their MFMAs) is left out of that run: each XCD takes its share of those cheap
  // tiles after its share of the others, so that they fill the last, partial round of tiles. Weight-gradient
  // tiles cost K = rows of their group, heaviest groups first (or, with wg_interleave, one tile of each group in
  // turn); they are dealt round-robin over the XCDs so that the long ones spread out.
  int L;
  bool tail = false;
  // Split tail tiles: the largest power of two up to tail_split whose windows of all tail tiles fit tail_cus
  // workgroups (a split tail tile takes about as long as a whole one, so more windows than CUs cost a round).
  int ts = 1;
  if (split && p.tail_split > 1) {
    const int ptiles = wave_pick(tl, G) * p.n_tiles;
    ts = p.tail_split;
    while (ts > 1 && ptiles * ts > p.tail_cus) ts >>= 1;
  }
  if (RAGGED) {
    // XCD x = bid % 8 takes the run [x * q + min(x, r), ...) of q or q + 1 tiles (total = 8 q + r) of each
    // segment: the counts differ by at most one between XCDs
    const int x = bid & 7, lb = bid >> 3;
    const int q = total >> 3, r = total & 7;
    const int cnt = q + (x < r ? 1 : 0);
    if (lb < cnt) {
      L = x * q + min(x, r) + lb;
    } else {
      if (!split) return false;
      const int ptot = wave_pick(tl, G) * p.n_tiles * ts;
      const int qt = ptot >> 3, rt = ptot & 7;
      const int lt = lb - cnt;
      if (lt >= qt + (x < rt ? 1 : 0)) return false;
      L = x * qt + min(x, rt) + lt;
      tail = true;
    }
  } else {
    L = bid;
  }
  if (!tail && L >= total) return false;
  int l, n_mt;
  t.sub = 0;
  t.nsub = 1;
  if (tail) {
    // the group of tail tile L / (n_tiles * ts): largest g whose tail prefix is <= it (groups without a tail share
    // their successor's prefix and are passed over); a split tail tile's windows are consecutive
    const int tix = L / (p.n_tiles * ts);
    int g = 0;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      if (s < ns) {
        const int i = 64 * s + lane;
        g += __popcll(__ballot(i >= 1 && i < G && tl[s] <= tix));
      }
    }
    g = __builtin_amdgcn_readfirstlane(g);
    t.g = g;
    const bool routed_t = g < p.Eloc;
    t.row0 = routed_t ? wave_pick(off, g) : 0;
    t.rows = routed_t ? wave_pick(off, g + 1) - t.row0 : p.T;
    const int rem = L - tix * p.n_tiles * ts;
    t.nt = __builtin_amdgcn_readfirstlane(rem / ts);
    t.sub = __builtin_amdgcn_readfirstlane(rem - (rem / ts) * ts);
    t.nsub = ts;
    t.mt = __builtin_amdgcn_readfirstlane(wave_pick(pre, g + 1) - wave_pick(pre, g));  // after the group's others
    return true;
  }
  if (RAGGED) {
    // largest g < G with pre[g] * n_tiles <= L (pre is non-decreasing from pre[0] = 0)
    int g = 0;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      if (s < ns) {
        const int i = 64 * s + lane;
        g += __popcll(__ballot(i >= 1 && i < G && pre[s] * p.n_tiles <= L));
      }
    }
    g = __builtin_amdgcn_readfirstlane(g);
    t.g = g;
    const int p0 = wave_pick(pre, g);
    l = L - p0 * p.n_tiles;
    n_mt = wave_pick(pre, g + 1) - p0;
  } else {
    int rank;
    if (p.wg_interleave && p.order && wave_pick(ord, G) != 0) {  // one tile of each group in turn, heaviest first
      rank = L % G;
      l = L / G;
    } else {                // heaviest groups first: their long K loops start early
      rank = L / (p.m_tiles * p.n_tiles);
      l = L - rank * p.m_tiles * p.n_tiles;
    }
    t.g = p.order ? wave_pick(ord, rank) : rank;
    n_mt = p.m_tiles;
  }
  const bool routed = t.g < p.Eloc;
  t.row0 = routed ? wave_pick(off, t.g) : 0;
  t.rows = routed ? wave_pick(off, t.g + 1) - t.row0 : p.T;
  const int mblk = l / (GROUP_M * p.n_tiles);
  const int rem = l - mblk * GROUP_M * p.n_tiles;
  const int gsz = min(GROUP_M, n_mt - mblk * GROUP_M);
  t.nt = __builtin_amdgcn_readfirstlane(rem / gsz);
  t.mt = __builtin_amdgcn_readfirstlane(mblk * GROUP_M + rem % gsz);
  return true;
}

// Tile plan of the row-ragged contractions (one workgroup of 512 threads: at most 511 groups): pre0, pre1 and
// pre2 = m-tile prefixes for bm0-, bm1- and bm2-row tiles; for bm1-row tiles also body1 = prefix of the m-tiles
// other than the tails and tail1 = prefix of the tails (a last m-tile holding at most bm1 / 2 rows); order =
// groups by decreasing row count (ties by index), and order[G] = 1 when all groups' row counts lie within 25% of
// the largest (0 otherwise). It also sets zero[0 .. nzero) to 0 (the tile counters of the launches that follow).
__global__ __launch_bounds__(512) void mtile_prefix_kernel(const int32_t* __restrict__ offsets, int Eloc, int S,
                                                           int Tn, int bm0, int bm1, int bm2,
                                                           int32_t* __restrict__ pre0, int32_t* __restrict__ pre1,
                                                           int32_t* __restrict__ body1, int32_t* __restrict__ tail1,
                                                           int32_t* __restrict__ pre2, int32_t* __restrict__ order,
                                                           int32_t* __restrict__ zero, int nzero);

// fp32 path (generic LDS-tiled MFMA 16x16x4 kernel)
hipError_t ffn_fwd_f32(const moe_desc& d, const void* x, const void* xp, const int32_t* offsets, const void* wg,
                       const void* wu, const void* wd, void* yp, void* saved, int32_t* pre, hipStream_t s);
hipError_t ffn_bwd_f32(const moe_desc& d, const void* x, const void* xp, const void* dy, const void* dyp,
                       const int32_t* offsets, const void* wg, const void* wu, const void* wd, const void* saved,
                       void* dxp, void* dwg, void* dwu, void* dwd, void* dgu, int32_t* pre, hipStream_t s);

}  // namespace pcmoe
