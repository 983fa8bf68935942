// Expert passes of Alg. 6 (ForwardExpert / BackwardExpert) as grouped bf16 GEMMs on CDNA4 MFMA.
//
// Same six contractions as the fp32 path (see grouped_gemm.h), built for gfx950:
//   * operands stream global -> LDS with direct-to-LDS buffer loads (16 bytes per lane, no VGPR
//     staging) through a STAGES-deep ring of LDS buffers, so STAGES-1 K-tiles are in flight while
//     the MFMAs consume one; rows past a group's end read as zeros through the buffer range check;
//   * K-contiguous operands sit in LDS as 128-byte rows with a 16-byte-chunk XOR swizzle and feed
//     v_mfma_f32_16x16x32_bf16 through pairs of ds_read_b64 (measured faster than ds_read_b128 on
//     gfx950 when odd lane groups read their upper half first);
//   * operands whose K is the slow dimension (W_down / W_{gate,up} in the input gradients, both
//     operands of the weight gradients) stay in their natural [k][mn] layout and are transposed on
//     the way into registers by ds_read_b64_tr_b16 (two reads per MFMA operand);
//   * 256 x 256 tiles with 16 wavefronts (4 x 4, 64 x 64 each) by default, 192 x 256 tiles with 8
//     wavefronts for a single-round down projection, 128 x 128 tiles with 4 when a side is not a multiple
//     of 256; for d_model >= 4096, a software-pipelined 256 x 256 tile with 4 wavefronts (one per SIMD,
//     128 x 128 each, accumulators in AGPRs, 32-deep K-tiles in a 4-stage ring) for every contraction but
//     the down projection (and for dX + dW_gate|up wherever the dX grid fills 8 rounds of the chip); fp32
//     accumulators, per-wave epilogue staged through LDS (fp32, or bf16 for plain stores) and written as
//     16-byte chunks (SwiGLU and its adjoint fused);
//   * tiles decoded on the device from a plan of m-tile prefixes (grouped_gemm.h); independent
//     contractions of the backward share one launch (gemm_bf16_pair_kernel);
//   * large launches claim their last eighth of tiles by ticket, so XCDs that run ahead take more of them;
//     the pipelined tile's weight gradients run in persistent workgroups (wg_persistent) that overlap each
//     finished tile's epilogue with the next tile's first loads;
//   * a group's last m-tile with at most half a tile of rows (a tail) still loads its whole B panel: on the
//     pipelined tile its wavefronts with at most 64 rows issue half the MFMAs, and a down projection of a few
//     rounds splits its tail tiles into column windows that spread over the idle CUs of its last round.
#include "grouped_gemm.h"

#include <algorithm>
#include <cstdlib>
#include <cstring>

namespace pcmoe {

typedef int int32x4 __attribute__((ext_vector_type(4)));
typedef short short4v __attribute__((ext_vector_type(4)));

// Buffer resource over [base, base + bytes): loads at offsets >= bytes return zeros.
__device__ __forceinline__ int32x4 make_rsrc(const void* base, uint32_t bytes) {
  struct {
    const void* p;
    uint32_t range;
    uint32_t cfg;
  } r = {base, bytes, 0x00020000u};
  int32x4 v = __builtin_bit_cast(int32x4, r);
  v.x = __builtin_amdgcn_readfirstlane(v.x);
  v.y = __builtin_amdgcn_readfirstlane(v.y);
  v.z = __builtin_amdgcn_readfirstlane(v.z);
  v.w = __builtin_amdgcn_readfirstlane(v.w);
  return v;
}

// 16 bytes per lane from the buffer at byte offset voff into LDS at lds_dst + 16 * lane. Written as
// inline assembly on purpose: through the builtin, the compiler sees an LDS store it cannot tell apart
// from the operand buffer being read, and waits for every outstanding load (vmcnt(0)) before the next
// LDS read, which serialises each K-tile's load latency with the previous tile's MFMAs. Completion is
// tracked by the explicit vmcnt waits of the main loop instead.
__device__ __forceinline__ uint32_t lds_addr(const char* p) {
  return __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)p);
}
__device__ __forceinline__ void dma16(int32x4 rsrc, uint32_t m0, int voff) {
  asm volatile(
      "s_mov_b32 m0, %0\n\t"
      "s_nop 0\n\t"
      "buffer_load_dwordx4 %1, %2, 0 offen lds"
      :
      : "s"(__builtin_amdgcn_readfirstlane(m0)), "v"(voff), "s"(rsrc)
      : "memory", "m0");
}

// K-contiguous tile rows of BK bf16 (BK = 64: 8 chunks of 16 bytes; BK = 32: 4 chunks): chunk c of row r
// lives at chunk c ^ kc_swz(r). With the two 8-byte halves read by alternating lane groups, 16 rows of
// one chunk column then cover every bank once per LDS pass. The swizzle depends on row bits 0..3 only,
// and every 16 rows are followed by 16 bytes of padding (kc_row): a fragment 16 rows further is then
// at the same lane address plus an immediate offset (16 * ROWB + 16) that the compiler cannot fuse
// with its neighbour's read into one ds_read2 (which would need register moves to split again).
template <int BK>
__device__ __forceinline__ int kc_swz(int r) {
  if (BK == 64) return (r & 7) ^ ((r >> 3) & 1);
  return (r >> 2) & 3;
}
template <int ROWB>
__device__ __forceinline__ int kc_row(int r) { return r * ROWB + 16 * (r >> 4); }
// K-major tile rows (R*2 bytes): 16-byte chunk c of k-row k lives at chunk c ^ mc_swz(k).
__device__ __forceinline__ int mc_swz(int k) { return ((k & 3) << 1) | (((k >> 3) & 1) << 3); }
// K-major tiles 256 wide read by 64-wide wave tiles use a padded layout instead: 512-byte rows two to
// a 1 KB direct-load block, each block followed by 32 bytes of padding, odd rows rotated by 8 chunks.
// The 8 rows one ds_read_b64_tr_b16 pass touches then fall on 8 distinct 32-byte bank groups, and a
// lane's address for fragment i and k-step kk is its fragment-0 address plus 32 i + 16896 kk.
constexpr int MK_BLOCK = 1056;
__device__ __forceinline__ int mk_row(int k) { return (k >> 1) * MK_BLOCK + (k & 1) * 512; }

// A K-contiguous operand fragment as two 8-byte reads. Lane groups with odd q read the upper half of
// their 16-byte chunk first, so that the 32 lanes of one LDS pass cover all banks; the MFMA then sees
// k-elements 4..7 before 0..3 in those lanes, and the partner operand is read in the same order.
__device__ __forceinline__ Chunk lds_kc_pair(const char* chunk, int q) {
  const int h = (q & 1) * 8;
  const uint2 a = *reinterpret_cast<const uint2*>(chunk + h);
  const uint2 b = *reinterpret_cast<const uint2*>(chunk + (8 - h));
  Chunk c;
  c.w[0] = a.x;
  c.w[1] = a.y;
  c.w[2] = b.x;
  c.w[3] = b.y;
  return c;
}

// The whole 16-byte chunk in one read, in k order (the pipelined one-wavefront-per-SIMD tiles).
__device__ __forceinline__ Chunk lds_kc_whole(const char* chunk) {
  const uint4 v = *reinterpret_cast<const uint4*>(chunk);
  Chunk c;
  c.w[0] = v.x;
  c.w[1] = v.y;
  c.w[2] = v.z;
  c.w[3] = v.w;
  return c;
}

__device__ __forceinline__ Chunk lds_tr_pair(const char* a0, const char* a1) {
  typedef __attribute__((address_space(3))) short4v* lp;
  short4v r0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lp)(a0));
  short4v r1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lp)(a1));
  Chunk c;
  c.w[0] = (uint32_t)(uint16_t)r0[0] | ((uint32_t)(uint16_t)r0[1] << 16);
  c.w[1] = (uint32_t)(uint16_t)r0[2] | ((uint32_t)(uint16_t)r0[3] << 16);
  c.w[2] = (uint32_t)(uint16_t)r1[0] | ((uint32_t)(uint16_t)r1[1] << 16);
  c.w[3] = (uint32_t)(uint16_t)r1[2] | ((uint32_t)(uint16_t)r1[3] << 16);
  return c;
}

// The same MFMA with its accumulator pinned to AGPRs and updated in place. With 256 accumulator registers per
// lane, the compiler's own choice writes some results to other registers and then moves every accumulator
// around the loop. Reads of the result by anything but the next MFMA on the same accumulator follow only after
// the K loop (and its trailing s_nops). Volatile: the MFMAs keep their order relative to the direct loads and
// barriers they are interleaved with (the scheduler would otherwise bunch the loads together).
__device__ __forceinline__ void mfma_bf16_agpr(floatx4& acc, const Chunk& a, const Chunk& b) {
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0"
      : "+a"(acc)
      : "v"(__builtin_bit_cast(int32x4, a)), "v"(__builtin_bit_cast(int32x4, b)));
}
__device__ __forceinline__ void mfma_bf16(floatx4& acc, const Chunk& a, const Chunk& b) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), acc, 0,
                                                0, 0);
}

// Logistic sigmoid for epilogues whose results are rounded to bf16: hardware exp and reciprocal (about
// 1 ulp of fp32 each) instead of an IEEE division; saturates to 0 and 1 at the tails.
__device__ __forceinline__ float sigmoid_bf16_out(float x) { return __builtin_amdgcn_rcpf(1.f + __expf(-x)); }

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

template <int BM, int BN, int BK, int STAGES, int WM, int WN>
struct Cfg2 {
  static constexpr int NW = WM * WN;
  static constexpr int NT = 64 * NW;
  static constexpr int WTM = BM / WM, WTN = BN / WN;
  static constexpr int FM = WTM / 16, FN = WTN / 16;
  static constexpr int ROWB = BK * 2;              // bytes of one K-contiguous tile row
  static constexpr int CR = ROWB / 16;             // 16-byte chunks per K-contiguous row
  static constexpr int RPI = 1024 / ROWB;          // K-contiguous rows per direct-load instruction
  static constexpr int KK = BK / 32;               // MFMA k-steps per K-tile
  // padding: 16 bytes per 16 K-contiguous rows, or 32 bytes per 1 KB block of a padded K-major tile
  static constexpr int PAD_A = (BM > 32 * (BM * ROWB / 1024) ? BM : 32 * (BM * ROWB / 1024));
  static constexpr int PAD_B = (BN > 32 * (BN * ROWB / 1024) ? BN : 32 * (BN * ROWB / 1024));
  static constexpr int A_BYTES = BM * ROWB + PAD_A;
  static constexpr int STAGE_BYTES = A_BYTES + BN * ROWB + PAD_B;
  static constexpr int LDS_MAIN = STAGES * STAGE_BYTES;
  static constexpr int PART_ROWS = WTM < 32 ? WTM : 32;
  static constexpr int PITCH = WTN + 4;  // fp32 epilogue staging pitch
  static constexpr int WAVE_EPI = PART_ROWS * PITCH * 4;
  static constexpr int LDS_EPI = NW * WAVE_EPI;
  static constexpr int LDS = LDS_MAIN > LDS_EPI ? LDS_MAIN : LDS_EPI;
  static constexpr int IA = BM * ROWB / 1024 / NW;  // direct loads per wave per K-tile (1 KB each)
  static constexpr int IB = BN * ROWB / 1024 / NW;
  static constexpr int LOADS = IA + IB;
  // 256 x 256 tiles with 4 wavefronts (one per SIMD, 128 x 128 each, 256 accumulator registers): the
  // software-pipelined K loop, and a kernel that may use all 512 registers of a lane
  static constexpr bool PIPE = NW == 4 && BM == 256 && BN == 256;
  static constexpr int WAVES_PER_EU = PIPE ? 1 : (NW >= 4 ? NW / 4 : 1);
  static_assert(IA * 1024 * NW == BM * ROWB && IB * 1024 * NW == BN * ROWB, "tiles must split evenly over waves");
};

// One output tile of contraction KIND: workgroup `bid` of that contraction's tile grid.
template <int BM, int BN, int BK, int KIND, int STAGES, int WM, int WN>
__device__ __forceinline__ void gemm_tile(const GemmArgs& p, int bid, char* smem) {
  using C = Cfg2<BM, BN, BK, STAGES, WM, WN>;
  using KT = KindTraits<KIND>;
  constexpr int ES = 2;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform (LDS DMA bases, resources)
  const int wm = wave / WN, wn = wave % WN;

  TileIdx ti;
  if (!decode_tile<KT::ragged_m>(p, bid, ti)) return;
  const int g = ti.g;
  const int d = p.d, f = p.f;
  const bool routed = g < p.Eloc;
  const int row0 = ti.row0, rows = ti.rows;
  const size_t rs = routed ? (size_t)row0 : (size_t)p.rows_cap + (size_t)(g - p.Eloc) * p.T;
  const int m0 = ti.mt * BM, n0 = ti.nt * BN;
  // A split tail tile of the down projection (two-stage ring) computes only the columns of its window: the other
  // wavefront columns skip their MFMAs and stores, and the B loads of the rows outside the window are not issued.
  // Every other tile is one window of the whole tile.
  const int nsub = (KIND == FWD_DOWN && STAGES == 2) ? ti.nsub : 1;
  const int wlo = ti.sub * (BN / nsub), whi = wlo + BN / nsub;
  int K;
  if (KIND == FWD_GU || KIND == BWD_DH) K = d;
  else if (KIND == FWD_DOWN) K = f;
  else if (KIND == BWD_DX) K = 2 * f;
  else K = rows;

  // ------------------------------------------------------------------ operand sources
  // A (M side). Ragged kinds: K-contiguous rows of the group; weight gradients: [rows][M] (K-major).
  // B (N side); B1: W_up (FWD_GU rows of the up half; BWD_DX K rows >= f). Each as a base and a byte range.
  const char *a_base, *b0_base, *b1_base;
  uint32_t a_bytes, b_bytes;
  int a_ld, b_ld;  // bytes between consecutive rows in memory
  if (KIND == FWD_GU) { a_base = routed ? (const char*)p.xp + rs * d * ES : (const char*)p.x; a_ld = d * ES; }
  else if (KIND == FWD_DOWN) { a_base = (const char*)p.h + rs * f * ES; a_ld = f * ES; }
  else if (KIND == BWD_DH || KIND == WG_DOWN) {
    a_base = routed ? (const char*)p.dyp + rs * d * ES : (const char*)p.dy;
    a_ld = d * ES;
  } else { a_base = (const char*)p.dgu + rs * 2 * f * ES; a_ld = 2 * f * ES; }
  a_bytes = (uint32_t)((size_t)rows * a_ld);
  if (KIND == FWD_GU || KIND == BWD_DX) {
    b0_base = (const char*)p.wg + (size_t)g * f * d * ES;
    b1_base = (const char*)p.wu + (size_t)g * f * d * ES;
    b_bytes = (uint32_t)((size_t)f * d * ES);
    b_ld = d * ES;
  } else if (KIND == FWD_DOWN || KIND == BWD_DH) {
    b0_base = b1_base = (const char*)p.wd + (size_t)g * d * f * ES;
    b_bytes = (uint32_t)((size_t)d * f * ES);
    b_ld = f * ES;
  } else if (KIND == WG_DOWN) {
    b0_base = b1_base = (const char*)p.h + rs * f * ES;
    b_bytes = (uint32_t)((size_t)rows * f * ES);
    b_ld = f * ES;
  } else {  // WG_GU
    b0_base = b1_base = routed ? (const char*)p.xp + rs * d * ES : (const char*)p.x;
    b_bytes = (uint32_t)((size_t)rows * d * ES);
    b_ld = d * ES;
  }
  const int32x4 ra = make_rsrc(a_base, a_bytes), rb0 = make_rsrc(b0_base, b_bytes), rb1 = make_rsrc(b1_base, b_bytes);

  // K-major operands in the padded layout (mk_row); a 128-wide wave tile reads two of its 64-column blocks
  constexpr bool MKP_A = !KT::a_kc && BM == 256 && (C::WTM == 64 || C::WTM == 128);
  constexpr bool MKP_B = !KT::b_kc && BN == 256 && (C::WTN == 64 || C::WTN == 128);

  // Per-lane byte offset at K-tile 0 of direct-load instruction jj (0 .. BM*ROWB/1024 - 1) of each operand;
  // for FWD_GU also whether the instruction's rows are W_up rows.
  const auto a_off = [&](int jj) {
    if (KT::a_kc) {
      const int r = C::RPI * jj + lane / C::CR, c = (lane % C::CR) ^ kc_swz<BK>(r);
      return (m0 + r) * a_ld + 16 * c;
    } else if (MKP_A) {
      const int kr = 2 * jj + (lane >> 5), c = ((lane & 31) - 8 * (kr & 1)) & 31;
      return kr * a_ld + (m0 + 8 * c) * ES;
    } else {
      constexpr int CPR = BM / 8;
      const int slot = 64 * jj + lane, kr = slot / CPR, c = (slot % CPR) ^ mc_swz(kr);
      return kr * a_ld + (m0 + 8 * c) * ES;
    }
  };
  const auto b_off = [&](int jj, bool& up) {
    up = false;
    if (KT::b_kc) {
      const int r = C::RPI * jj + lane / C::CR, c = (lane % C::CR) ^ kc_swz<BK>(r);
      int wrow;
      if (KIND == FWD_GU) {
        const int wcol = r / C::WTN, within = r % C::WTN, half = C::WTN / 2;
        static_assert((C::WTN / 2) % C::RPI == 0, "a direct load must not straddle gate and up rows");
        wrow = ti.nt * (BN / 2) + wcol * half + (within % half);
        up = ((C::RPI * jj) % C::WTN) >= half;  // the instruction's rows are all gate or all up rows
      } else {
        wrow = n0 + r;
      }
      return wrow * b_ld + 16 * c;
    } else if (MKP_B) {
      const int kr = 2 * jj + (lane >> 5), c = ((lane & 31) - 8 * (kr & 1)) & 31;
      return kr * b_ld + (n0 + 8 * c) * ES;
    } else {
      constexpr int CPR = BN / 8;
      const int slot = 64 * jj + lane, kr = slot / CPR, c = (slot % CPR) ^ mc_swz(kr);
      return kr * b_ld + (n0 + 8 * c) * ES;
    }
  };
  // LDS padding before instruction jj: K-contiguous rows RPI * jj .. RPI * jj + RPI - 1 follow 16 bytes per
  // earlier 16 rows; a padded K-major block follows 32 bytes per earlier block
  const auto pad = [&](int jj, bool kc, bool mkp) { return kc ? 16 * ((C::RPI * jj) >> 4) : (mkp ? 32 * jj : 0); };
  const uint32_t lds_base = lds_addr(smem);
  // Direct load of instruction jj of operand A (or B) of K-tile kt into LDS stage `stage`.
  const auto load_a = [&](int kt, int stage, int jj, int voff) {
    // Row-ragged tiles in a two-stage ring (whose waits are vmcnt(0)): an instruction whose rows all lie past the
    // group's end is skipped; those rows' outputs are never stored, and no other row reads them.
    if (KT::ragged_m && STAGES == 2 && m0 + C::RPI * jj >= rows) return;
    const int k0 = kt * BK;
    dma16(ra, lds_base + stage * C::STAGE_BYTES + jj * 1024 + pad(jj, KT::a_kc, MKP_A),
          voff + (KT::a_kc ? k0 * ES : k0 * a_ld));
  };
  const auto load_b = [&](int kt, int stage, int jj, int voff, bool up) {
    // (a split tail tile: every row of instruction jj lies outside the window or none does; the waits are vmcnt(0))
    if (KIND == FWD_DOWN && STAGES == 2 && (C::RPI * jj < wlo || C::RPI * jj >= whi)) return;
    const int k0 = kt * BK;
    const uint32_t dst = lds_base + stage * C::STAGE_BYTES + C::A_BYTES + jj * 1024 + pad(jj, KT::b_kc, MKP_B);
    if (KIND == BWD_DX) {
      const bool hi = k0 >= f;  // K rows >= f are W_up rows
      dma16(hi ? rb1 : rb0, dst, voff + (hi ? k0 - f : k0) * b_ld);
    } else {
      dma16(up ? rb1 : rb0, dst, voff + (KT::b_kc ? k0 * ES : k0 * b_ld));
    }
  };

  floatx4 acc[C::FM][C::FN];
#pragma unroll
  for (int i = 0; i < C::FM; ++i)
#pragma unroll
    for (int j = 0; j < C::FN; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  const int KTN = (K + BK - 1) / BK;
  const int q = lane >> 4, li = lane & 15;
  const bool wave_rows = !KT::ragged_m || m0 + wm * C::WTM < rows;  // wave-uniform
  // The last n-tile of a contraction whose N is not a multiple of BN holds fewer columns (N is a multiple of
  // 128 and a wave's columns a 64-aligned block, so each wave's columns are all inside or all past N). Its
  // B loads past N read neighbouring rows or zeros through the buffer range check: finite values that reach
  // only the columns past N, which are neither computed nor stored.
  const bool wave_cols = n0 + wn * C::WTN < p.n_extent && wn * C::WTN >= wlo && wn * C::WTN < whi;  // wave-uniform

  // Operand fragments of MFMA k-step kk (32 deep) of the K-tile whose stage starts at As (A) / Bs (B).
  // K-contiguous fragments: row 16 * i + li of the wave's rows; the swizzle sees only li, and fragment i sits FRAG
  // bytes after fragment 0 (an immediate offset of the LDS read). Odd lane groups take k-elements 4..7 before
  // 0..3 (lds_kc_pair), and the transposed reads of the partner operand follow the same order (SW = 1); with it
  // the transposed reads of the padded layout hit 8 distinct bank groups per pass. The pipelined tiles read a
  // K-contiguous fragment whole and in k order (SW = 0: one LDS instruction per fragment, which measured faster
  // there), at the cost of 2-way bank conflicts in the transposed reads of the contractions that mix both kinds.
  constexpr int FRAG = 16 * C::ROWB + 16;
  constexpr int SW = (C::PIPE && (KT::a_kc || KT::b_kc)) ? 0 : 1;
  // padded K-major fragments: the lane's two k-rows (kl1, kl2) and its 8-byte column group; fragment i of a wave
  // tile lies in 64-column block (wave offset + 16 i) / 64, at 32 (i mod 4) bytes
  const int kl1 = 8 * q + 4 * SW * (q & 1) + (li >> 2), kl2 = kl1 + 4 - 8 * SW * (q & 1);
  const auto mk_lane = [&](int kl, int w, int kk) {
    return mk_row(kl) + 128 * ((w + (kl & 1)) & 3) + 16 * ((li & 3) >> 1) + 8 * (li & 1) + 16 * MK_BLOCK * kk;
  };
  const auto frag_a = [&](const char* As, int kk, int i) {
    if (KT::a_kc) {
      const int lane_kc = li * C::ROWB + (((4 * kk + q) ^ kc_swz<BK>(li)) << 4);
      const char* ch = As + kc_row<C::ROWB>(wm * C::WTM) + lane_kc + i * FRAG;
      return C::PIPE ? lds_kc_whole(ch) : lds_kc_pair(ch, q);
    } else if (MKP_A) {
      const int w = (wm * C::WTM) / 64 + i / 4;
      return lds_tr_pair(As + mk_lane(kl1, w, kk) + 32 * (i % 4), As + mk_lane(kl2, w, kk) + 32 * (i % 4));
    } else {
      const int k1 = 32 * kk + kl1, k2 = 32 * kk + kl2, mn = wm * C::WTM + 16 * i + 4 * (li & 3);
      return lds_tr_pair(As + k1 * (BM * 2) + (((mn >> 3) ^ mc_swz(k1)) << 4) + (mn & 7) * 2,
                         As + k2 * (BM * 2) + (((mn >> 3) ^ mc_swz(k2)) << 4) + (mn & 7) * 2);
    }
  };
  const auto frag_b = [&](const char* Bs, int kk, int j) {
    if (KT::b_kc) {
      const int lane_kc = li * C::ROWB + (((4 * kk + q) ^ kc_swz<BK>(li)) << 4);
      const char* ch = Bs + kc_row<C::ROWB>(wn * C::WTN) + lane_kc + j * FRAG;
      return C::PIPE ? lds_kc_whole(ch) : lds_kc_pair(ch, q);
    } else if (MKP_B) {
      const int w = (wn * C::WTN) / 64 + j / 4;
      return lds_tr_pair(Bs + mk_lane(kl1, w, kk) + 32 * (j % 4), Bs + mk_lane(kl2, w, kk) + 32 * (j % 4));
    } else {
      const int k1 = 32 * kk + kl1, k2 = 32 * kk + kl2, mn = wn * C::WTN + 16 * j + 4 * (li & 3);
      return lds_tr_pair(Bs + k1 * (BN * 2) + (((mn >> 3) ^ mc_swz(k1)) << 4) + (mn & 7) * 2,
                         Bs + k2 * (BN * 2) + (((mn >> 3) ^ mc_swz(k2)) << 4) + (mn & 7) * 2);
    }
  };
  const auto read_frags = [&](const char* As, const char* Bs, int kk, Chunk (&a)[C::FM], Chunk (&b)[C::FN]) {
#pragma unroll
    for (int i = 0; i < C::FM; ++i) a[i] = frag_a(As, kk, i);
#pragma unroll
    for (int j = 0; j < C::FN; ++j) b[j] = frag_b(Bs, kk, j);
  };

  // Every wave loads IA + IB instructions of each K-tile (instruction jj = wave + NW j) and reads its fragments
  // one 32-deep k-step at a time; loads run one K-tile ahead of the MFMAs.
  int va[C::IA], vb[C::IB];
  bool bup[C::IB];
#pragma unroll
  for (int j = 0; j < C::IA; ++j) va[j] = a_off(wave + C::NW * j);
#pragma unroll
  for (int j = 0; j < C::IB; ++j) vb[j] = b_off(wave + C::NW * j, bup[j]);
  auto issue = [&](int kt, int stage) {
#pragma unroll
    for (int j = 0; j < C::IA; ++j) load_a(kt, stage, wave + C::NW * j, va[j]);
#pragma unroll
    for (int j = 0; j < C::IB; ++j) load_b(kt, stage, wave + C::NW * j, vb[j], bup[j]);
  };
  if constexpr (C::PIPE) {
    // One wavefront per SIMD (4 wavefronts of 128 x 128): no other wavefront hides a stall of this one, so the
    // K loop is software-pipelined by hand. 32-deep K-tiles in a 4-stage ring; a K-tile's fragments are read into
    // registers during the step before the one that multiplies them, so its stage is free again from that step's
    // end. In the step of K-tile kt:
    //   * MFMAs 0..15 of kt;
    //   * the wait for this wave's loads of K-tile kt + 1 and a workgroup barrier: every wave's loads of kt + 1
    //     have landed, and every wave has read K-tile kt (so its stage is free);
    //   * MFMAs 16..63 of kt, with the 16 fragment reads of kt + 1 (into the other register set, in the order the
    //     next step uses them) and the 8 direct loads of K-tile kt + 4 (into kt's stage) between them.
    // A load has three steps to land before the barrier that waits for it.
    // Every instruction of the step keeps this order (the MFMAs and the loads are volatile asm, the reads cannot
    // cross them). Nothing in the step branches: a branch around MFMAs makes the compiler copy all 256
    // accumulators. So the loop runs an even number of steps (K-tiles past K are zeros: only the weight
    // gradients, whose K rows end at the group's end, can have an odd count), and the loads of K-tiles past the
    // last one are issued with an offset past every buffer range (they return zeros and fetch nothing). A
    // wavefront with no rows or no columns to compute takes the same loads and barriers without MFMAs and
    // fragment reads, and then returns.
    static_assert(STAGES == 4 && C::KK == 1 && C::IA == 4 && C::IB == 4 && C::FM == 8 && C::FN == 8,
                  "pipelined tile");
    const int KTN2 = (KTN + 1) & ~1;
    constexpr int OOR = 0x7fffffff;  // no operand range reaches 2^31 bytes
    // load l (0..7, a constant after unrolling) of K-tile kt: one direct load whatever kt, so that nothing branches
    const auto load_one = [&](int kt, int l) {
      const bool live = kt < KTN;
      const int k0 = kt * BK;
      const uint32_t st = lds_base + (kt & 3) * C::STAGE_BYTES;
      if (l < C::IA) {
        const int jj = wave + C::NW * l;
        const int off = va[l & (C::IA - 1)] + (KT::a_kc ? k0 * ES : k0 * a_ld);
        dma16(ra, st + jj * 1024 + pad(jj, KT::a_kc, MKP_A), live ? off : OOR);
      } else {
        const int j = (l - C::IA) & (C::IB - 1), jj = wave + C::NW * j;
        int off;
        int32x4 rsrc;
        if (KIND == BWD_DX) {
          const bool hi = k0 >= f;  // K rows >= f are W_up rows
          rsrc = hi ? rb1 : rb0;
          off = vb[j] + (hi ? k0 - f : k0) * b_ld;
        } else {
          rsrc = bup[j] ? rb1 : rb0;
          off = vb[j] + (KT::b_kc ? k0 * ES : k0 * b_ld);
        }
        dma16(rsrc, st + C::A_BYTES + jj * 1024 + pad(jj, KT::b_kc, MKP_B), live ? off : OOR);
      }
    };
    const auto issue_all = [&](int kt) {
#pragma unroll
      for (int l = 0; l < 8; ++l) load_one(kt, l);
    };
    const auto barrier = [] { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); };
    issue_all(0);
    issue_all(1);
    issue_all(2);
    issue_all(3);
    wait_vmcnt<24>();  // K-tile 0 has landed
    barrier();
    if (!wave_rows || !wave_cols) {
      for (int kt = 0; kt < KTN2; ++kt) {
        wait_vmcnt<16>();  // K-tile kt + 1 has landed (kt + 2 and kt + 3 may be in flight)
        barrier();
        issue_all(kt + 4);
      }
      wait_vmcnt<0>();
      __syncthreads();
      return;
    }
    Chunk fa[2][C::FM], fb[2][C::FN];
    read_frags(smem, smem + C::A_BYTES, 0, fa[0], fb[0]);
    // The step of K-tile kt with its fragments in register set S, for the first FMA row blocks of the wavefront:
    // all 8, or 4 when its rows past the first 64 all lie past the group's end (a group's last m-tile; the MFMAs
    // of the empty blocks would leave their accumulators at zero, and the epilogue skips those rows). The half
    // step spreads the same fragment reads of its blocks and the same 8 direct loads over its 24 MFMAs after the
    // barrier, so the waits and barriers are those of the full step.
    const auto step = [&](int kt, auto set, auto blocks) {
      constexpr int S = decltype(set)::value;
      constexpr int FMA = decltype(blocks)::value;
      constexpr int NM = FMA * C::FN;                // MFMAs of the step
      constexpr int MB = NM / 4;                     // MFMAs before the wait and barrier
      constexpr int RS = (NM - MB) / (FMA + C::FN);  // MFMAs per fragment read: 3, or 2 for the half step
      constexpr int LS = (NM - MB) / 8;              // MFMAs per direct load: 6, or 3
      static_assert(RS * (FMA + C::FN) == NM - MB && LS * 8 == NM - MB, "pipelined step schedule");
      const char* As = smem + ((kt + 1) & 3) * C::STAGE_BYTES;
#pragma unroll
      for (int i = 0; i < FMA; ++i) {
#pragma unroll
        for (int j = 0; j < C::FN; ++j) {
          const int m = i * C::FN + j;
          if (m == MB) {
            wait_vmcnt<16>();  // K-tile kt + 1 has landed (kt + 2 and kt + 3 may be in flight)
            barrier();
          }
          mfma_bf16_agpr(acc[i][j], fb[S][j], fa[S][i]);  // transposed block: 4 consecutive columns per lane
          if (m >= MB) {
            const int r = m - MB;  // a read after every RS-th MFMA, a load after every LS-th
            if (r % RS == 0) {
              const int t = r / RS;  // fa[0], fb[0..7], fa[1..FMA-1]
              if (t == 0) fa[S ^ 1][0] = frag_a(As, 0, 0);
              else if (t <= C::FN) fb[S ^ 1][t - 1] = frag_b(As + C::A_BYTES, 0, t - 1);
              else fa[S ^ 1][t - C::FN] = frag_a(As, 0, t - C::FN);
            }
            if (r % LS == LS / 3) load_one(kt + 4, r / LS);
          }
        }
      }
    };
    if (KT::ragged_m && m0 + wm * C::WTM + C::WTM / 2 >= rows) {  // wave-uniform
      for (int kt = 0; kt < KTN2; kt += 2) {
        step(kt, std::integral_constant<int, 0>{}, std::integral_constant<int, C::FM / 2>{});
        step(kt + 1, std::integral_constant<int, 1>{}, std::integral_constant<int, C::FM / 2>{});
      }
    } else {
      for (int kt = 0; kt < KTN2; kt += 2) {
        step(kt, std::integral_constant<int, 0>{}, std::integral_constant<int, C::FM>{});
        step(kt + 1, std::integral_constant<int, 1>{}, std::integral_constant<int, C::FM>{});
      }
    }
    wait_vmcnt<0>();  // the zero-filling loads past the last K-tile land before the epilogue reuses the LDS
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");  // the last MFMAs' results are ready to read
  } else {
  // prologue: STAGES-1 tiles in flight
#pragma unroll
  for (int s = 0; s < STAGES - 1; ++s)
    if (s < KTN) issue(s, s);
  for (int kt = 0; kt < KTN; ++kt) {
    // tile kt has landed when at most the later tiles' loads are outstanding
    if (kt + STAGES - 2 < KTN) wait_vmcnt<(STAGES - 2) * C::LOADS>();
    else wait_vmcnt<0>();
    // every wave's loads of tile kt have landed and its reads of the stage about to be refilled are done
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    if (kt + STAGES - 1 < KTN) issue(kt + STAGES - 1, (kt + STAGES - 1) % STAGES);
    // a wavefront whose rows all lie past the group's end, or whose columns all lie past N, has nothing to
    // compute (it still loads and syncs)
    if (!wave_rows || !wave_cols) continue;
    const char* As = smem + (kt % STAGES) * C::STAGE_BYTES;
    const char* Bs = As + C::A_BYTES;
#pragma unroll
    for (int kk = 0; kk < C::KK; ++kk) {
      Chunk a[C::FM], b[C::FN];
      read_frags(As, Bs, kk, a, b);
#pragma unroll
      for (int i = 0; i < C::FM; ++i)
#pragma unroll
        for (int j = 0; j < C::FN; ++j) mfma_bf16(acc[i][j], a[i], b[j]);
    }
  }
  }
  __syncthreads();  // every wave is done with the operand buffers

  // ------------------------------------------------------------------ epilogue (per wave)
  if (!wave_cols) return;  // no output column of this wave lies inside N (the epilogue has no workgroup barrier)
  float* st = reinterpret_cast<float*>(smem + wave * C::WAVE_EPI);
  constexpr int FPP = C::PART_ROWS / 16;  // fm blocks per part
  constexpr int OUT_W = (KIND == FWD_GU) ? C::WTN / 2 : C::WTN;  // output columns of the wave
  constexpr int CPRW = OUT_W / 8;                                  // 16-byte output chunks per row
  if constexpr (C::PIPE && (KIND == BWD_DX || KIND == WG_DOWN || KIND == WG_GU)) {
    // Plain stores of the pipelined tile: each lane rounds its four consecutive columns of a block to bf16 (the
    // rounding the fp32 staging would apply on the way out) and stages them with one 8-byte write; the 16-byte
    // output chunks are then read whole. Rows of 128 + 8 bf16 keep both sides free of bank conflicts.
    constexpr int P16 = C::WTN + 8;
    char* sb = smem + wave * C::WAVE_EPI;
#pragma unroll
    for (int part = 0; part < C::FM / FPP; ++part) {
#pragma unroll
      for (int i = 0; i < FPP; ++i)
#pragma unroll
        for (int j = 0; j < C::FN; ++j) {
          const floatx4 v = acc[part * FPP + i][j];
          uint2 pk;
          pk.x = pack_bf16x2(v[0], v[1]);
          pk.y = pack_bf16x2(v[2], v[3]);
          *reinterpret_cast<uint2*>(sb + ((16 * i + li) * P16 + 16 * j + 4 * q) * 2) = pk;
        }
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // this wave's staging writes are done
      __builtin_amdgcn_wave_barrier();
      for (int qq = lane; qq < C::PART_ROWS * CPRW; qq += 64) {
        const int rr = qq / CPRW, cc = (qq % CPRW) * 8;
        const int m = m0 + wm * C::WTM + part * C::PART_ROWS + rr;
        if (KT::ragged_m && m >= rows) continue;
        const Chunk v = *reinterpret_cast<const Chunk*>(sb + (rr * P16 + cc) * 2);
        if (KIND == BWD_DX) {
          st_chunk((char*)p.out + ((rs + m) * d + n0 + wn * OUT_W + cc) * ES, v);
        } else if (KIND == WG_DOWN) {
          st_chunk_nt((char*)p.out + (((size_t)g * d + m) * f + n0 + wn * OUT_W + cc) * ES, v);
        } else {  // WG_GU
          const int col = n0 + wn * OUT_W + cc;
          char* o = (m < f) ? (char*)p.out + (((size_t)g * f + m) * d + col) * ES
                            : (char*)p.out2 + (((size_t)g * f + (m - f)) * d + col) * ES;
          st_chunk_nt(o, v);
        }
      }
      __builtin_amdgcn_wave_barrier();
    }
    return;
  }
  // The SwiGLU adjoint (BWD_DH) reads the saved G|U of its outputs. The pipelined tile's wavefronts have four times
  // the outputs of a 16-wavefront tile's, so there the loads of the next part are issued before this part is
  // staged and computed (two register buffers), and their latency is paid about once per tile instead of per part.
  constexpr int GU_IT = C::PART_ROWS * CPRW / 64;  // output chunks per lane and part
  constexpr bool GU_AHEAD = KIND == BWD_DH && C::PIPE;
  Chunk gbuf[GU_AHEAD ? 2 : 1][GU_IT], ubuf[GU_AHEAD ? 2 : 1][GU_IT];
  const auto load_gu = [&](int part, Chunk (&gch)[GU_IT], Chunk (&uch)[GU_IT]) {
#pragma unroll
    for (int it = 0; it < GU_IT; ++it) {
      const int qq = lane + 64 * it, rr = qq / CPRW, cc = (qq % CPRW) * 8;
      const int m = min(m0 + wm * C::WTM + part * C::PART_ROWS + rr, rows - 1);  // rows past the group: unused
      const char* gu = (const char*)p.gu + ((rs + m) * 2 * f + n0 + wn * OUT_W + cc) * ES;
      gch[it] = ld_chunk(gu);
      uch[it] = ld_chunk(gu + (size_t)f * ES);
    }
  };
  if constexpr (GU_AHEAD) load_gu(0, gbuf[0], ubuf[0]);
#pragma unroll
  for (int part = 0; part < C::FM / FPP; ++part) {
    if constexpr (GU_AHEAD) {
      if (part + 1 < C::FM / FPP) load_gu(part + 1, gbuf[(part + 1) & 1], ubuf[(part + 1) & 1]);
    }
    if constexpr (C::PIPE) {
      // The pipelined tile multiplies B by A: lane (q, li) of block (i, j) holds row 16 i + li, columns 16 j + 4 q ..
      // 16 j + 4 q + 3, staged with one 16-byte write.
#pragma unroll
      for (int i = 0; i < FPP; ++i)
#pragma unroll
        for (int j = 0; j < C::FN; ++j)
          *reinterpret_cast<floatx4*>(st + (16 * i + li) * C::PITCH + 16 * j + 4 * q) = acc[part * FPP + i][j];
    } else {
#pragma unroll
      for (int i = 0; i < FPP; ++i)
#pragma unroll
        for (int j = 0; j < C::FN; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r) st[(16 * i + 4 * q + r) * C::PITCH + 16 * j + li] = acc[part * FPP + i][j][r];
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // this wave's staging writes are done
    __builtin_amdgcn_wave_barrier();
    if constexpr (KIND == BWD_DH) {
      // (the 16-wavefront tiles load the whole part's G|U together here, so their latency is paid once per part)
      constexpr int IT = GU_IT;
      static_assert(IT * 64 == C::PART_ROWS * CPRW, "epilogue chunks per lane");
      Chunk(&gch)[IT] = gbuf[GU_AHEAD ? (part & 1) : 0];
      Chunk(&uch)[IT] = ubuf[GU_AHEAD ? (part & 1) : 0];
      if constexpr (!GU_AHEAD) load_gu(part, gch, uch);
#pragma unroll
      for (int it = 0; it < IT; ++it) {
        const int qq = lane + 64 * it, rr = qq / CPRW, cc = (qq % CPRW) * 8;
        const int m = m0 + wm * C::WTM + part * C::PART_ROWS + rr;
        if (m >= rows) continue;
        float v[8], gv[8], uv[8], dg[8], du[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = st[rr * C::PITCH + cc + e];
        chunk_to_f<bf16>(gch[it], gv);
        chunk_to_f<bf16>(uch[it], uv);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float sg = sigmoid_bf16_out(gv[e]);
          du[e] = v[e] * gv[e] * sg;
          dg[e] = v[e] * uv[e] * sg * (1.f + gv[e] * (1.f - sg));
        }
        char* o = (char*)p.dgu + ((rs + m) * 2 * f + n0 + wn * OUT_W + cc) * ES;
        st_chunk(o, f_to_chunk<bf16>(dg));
        st_chunk(o + (size_t)f * ES, f_to_chunk<bf16>(du));
      }
      __builtin_amdgcn_wave_barrier();
      continue;
    }
    for (int qq = lane; qq < C::PART_ROWS * CPRW; qq += 64) {
      const int rr = qq / CPRW, cc = (qq % CPRW) * 8;
      const int m = m0 + wm * C::WTM + part * C::PART_ROWS + rr;
      if (KT::ragged_m && m >= rows) continue;
      float v[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = st[rr * C::PITCH + cc + e];
      if (KIND == FWD_GU) {
        float u[8], hv[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          u[e] = st[rr * C::PITCH + OUT_W + cc + e];
          const float sg = sigmoid_bf16_out(v[e]);
          hv[e] = v[e] * sg * u[e];
        }
        const int col = ti.nt * (BN / 2) + wn * OUT_W + cc;
        char* gu = (char*)p.gu + ((rs + m) * 2 * f + col) * ES;
        st_chunk(gu, f_to_chunk<bf16>(v));
        st_chunk(gu + (size_t)f * ES, f_to_chunk<bf16>(u));
        st_chunk((char*)p.h + ((rs + m) * f + col) * ES, f_to_chunk<bf16>(hv));
      } else if (KIND == FWD_DOWN || KIND == BWD_DX) {
        st_chunk((char*)p.out + ((rs + m) * d + n0 + wn * OUT_W + cc) * ES, f_to_chunk<bf16>(v));
      } else if (KIND == WG_DOWN) {
        st_chunk_nt((char*)p.out + (((size_t)g * d + m) * f + n0 + wn * OUT_W + cc) * ES, f_to_chunk<bf16>(v));
      } else {  // WG_GU
        const int col = n0 + wn * OUT_W + cc;
        char* o = (m < f) ? (char*)p.out + (((size_t)g * f + m) * d + col) * ES
                          : (char*)p.out2 + (((size_t)g * f + (m - f)) * d + col) * ES;
        st_chunk_nt(o, f_to_chunk<bf16>(v));
      }
    }
    __builtin_amdgcn_wave_barrier();
  }
}

template <int BM, int BN, int BK, int KIND, int STAGES, int WM, int WN>
__global__ __launch_bounds__(64 * WM * WN) __attribute__((amdgpu_waves_per_eu(
    Cfg2<BM, BN, BK, STAGES, WM, WN>::WAVES_PER_EU))) void gemm_bf16_kernel(GemmArgs p, int dyn_first, int dyn) {
  extern __shared__ __align__(16) char smem[];
  __shared__ int ticket;
  const int bid = blockIdx.x;
  if (bid < dyn_first) {
    gemm_tile<BM, BN, BK, KIND, STAGES, WM, WN>(p, bid, smem);
  } else {  // ticket-claimed: workgroup index dyn_first + ticket of the static grid (see gemm_bf16_pair_kernel)
    if (threadIdx.x == 0) ticket = __hip_atomic_fetch_add(p.tickets, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    const int t = ticket;
    if (t < dyn) gemm_tile<BM, BN, BK, KIND, STAGES, WM, WN>(p, dyn_first + t, smem);
  }
}

// Weight-gradient tiles of the pipelined 256 x 256 shape in persistent workgroups (one per CU), for the second
// contraction of a paired launch. Tile L belongs to XCD L mod 8 (the static mapping's L2 locality); each XCD's
// workgroups take its tiles in order from a counter of their own, and take another XCD's once theirs run out.
// Per tile, after the K loop: the next tile is decoded (from plan arrays loaded once, so without a memory round
// trip), its first four K-tiles are issued into the operand ring, and
// only then is the finished tile written out, through a staging area past the ring (16-row parts, bf16) that no load
// touches. The next K loop starts once every load and store has completed (vmcnt(0)), so no wait count ever spans
// stores. A tile is claimed one tile ahead from the workgroup's own XCD counter (the increment is issued with the
// prologue loads and its result read after the next K loop); only when that share is exhausted are the other XCDs'
// counters tried, one after the other. The loop ends when every counter is past its XCD's share, so every
// wavefront leaves.
constexpr int WG_STG_ROWS = 16;                              // staging rows per part
constexpr int WG_STG_WAVE = WG_STG_ROWS * (128 + 8) * 2;         // one wavefront's staging area (bf16)
constexpr int WG_LDS = Cfg2<256, 256, 32, 4, 2, 2>::LDS_MAIN + 4 * WG_STG_WAVE;
struct WgTile {
  int g, m0, n0, rows;
  size_t rs;
  bool cols;  // this wavefront's columns lie inside N
};
// Tile for claim result t of XCD x's counter, or -1 past x's share (tiles L = x, x + 8, ...).
__device__ __forceinline__ int wg_tile_of(int t, int x, int n_tiles) {
  return t >= 0 && t < ((n_tiles - x + 7) >> 3) ? 8 * t + x : -1;
}
// The other XCDs' counters in turn (lane 0 of wave 0 only): tile L, or -1 once every share is taken.
__device__ __forceinline__ int wg_steal(int* queues, int xcc, int n_tiles) {
  for (int i = 1; i < 8; ++i) {
    const int x = (xcc + i) & 7;
    const int L = wg_tile_of(__hip_atomic_fetch_add(queues + x, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT), x,
                             n_tiles);
    if (L >= 0) return L;
  }
  return -1;
}

template <int KIND>
__device__ __forceinline__ void wg_persistent(const GemmArgs& p, char* smem, int* queues, int n_tiles) {
  static_assert(KIND == WG_DOWN || KIND == WG_GU, "weight gradients only");
  using C = Cfg2<256, 256, 32, 4, 2, 2>;
  constexpr int ES = 2;
  constexpr int STG_ROWS = WG_STG_ROWS, P16 = C::WTN + 8, STG_WAVE = WG_STG_WAVE;
  static_assert(STG_WAVE == STG_ROWS * P16 * 2 && WG_LDS <= 160 * 1024, "ring and staging share the LDS");
  __shared__ int next_tile;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / 2, wn = wave % 2;
  const int q = lane >> 4, li = lane & 15;
  const int d = p.d, f = p.f;
  const int xcc = (int)(__builtin_amdgcn_s_getreg((3 << 11) | 20) & 7);  // HW_REG_XCC_ID
  const uint32_t lds_base = lds_addr(smem);
  char* stg = smem + C::LDS_MAIN + wave * STG_WAVE;

  if (tid == 0) {
    int L0 = wg_tile_of(__hip_atomic_fetch_add(queues + xcc, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT), xcc,
                        n_tiles);
    next_tile = L0 >= 0 ? L0 : wg_steal(queues, xcc, n_tiles);
  }
  __syncthreads();
  const int L = next_tile;
  if (L < 0) return;

  // the plan arrays of the decode, loaded once for every tile of the loop
  DecodeArrays plan;
  decode_load<false>(p, plan);
  // per-tile operand state
  int32x4 ra, rb;
  int a_ld, b_ld, va[4], vb[4], KTN = 0;
  WgTile cur;
  const auto setup = [&](int tile, WgTile& w) {
    TileIdx ti;
    decode_with<false>(p, tile, plan, ti);
    w.g = ti.g;
    const bool routed = ti.g < p.Eloc;
    w.rows = ti.rows;
    w.rs = routed ? (size_t)ti.row0 : (size_t)p.rows_cap + (size_t)(ti.g - p.Eloc) * p.T;
    w.m0 = ti.mt * 256;
    w.n0 = ti.nt * 256;
    w.cols = w.n0 + wn * C::WTN < p.n_extent;
    const char *a_base, *b_base;
    if (KIND == WG_DOWN) {
      a_base = routed ? (const char*)p.dyp + w.rs * d * ES : (const char*)p.dy;
      a_ld = d * ES;
      b_base = (const char*)p.h + w.rs * f * ES;
      b_ld = f * ES;
    } else {
      a_base = (const char*)p.dgu + w.rs * 2 * f * ES;
      a_ld = 2 * f * ES;
      b_base = routed ? (const char*)p.xp + w.rs * d * ES : (const char*)p.x;
      b_ld = d * ES;
    }
    ra = make_rsrc(a_base, (uint32_t)((size_t)w.rows * a_ld));
    rb = make_rsrc(b_base, (uint32_t)((size_t)w.rows * b_ld));
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int jj = wave + 4 * j;
      const int kr = 2 * jj + (lane >> 5), c = ((lane & 31) - 8 * (kr & 1)) & 31;
      va[j] = kr * a_ld + (w.m0 + 8 * c) * ES;
      vb[j] = kr * b_ld + (w.n0 + 8 * c) * ES;
    }
    KTN = (w.rows + 31) / 32;
  };
  constexpr int OOR = 0x7fffffff;
  const auto load_one = [&](int kt, int l) {
    const bool live = kt < KTN;
    const int k0 = kt * 32;
    const uint32_t st = lds_base + (kt & 3) * C::STAGE_BYTES;
    const int jj = wave + 4 * (l & 3);
    if (l < 4) dma16(ra, st + jj * 1024 + 32 * jj, live ? va[l & 3] + k0 * a_ld : OOR);
    else dma16(rb, st + C::A_BYTES + jj * 1024 + 32 * jj, live ? vb[l & 3] + k0 * b_ld : OOR);
  };
  const auto issue_all = [&](int kt) {
#pragma unroll
    for (int l = 0; l < 8; ++l) load_one(kt, l);
  };
  const auto barrier = [] { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); };
  // transposed fragment reads of the padded K-major layout (both operands), k order swapped in odd lane groups
  const int kl1 = 8 * q + 4 * (q & 1) + (li >> 2), kl2 = kl1 + 4 - 8 * (q & 1);
  const auto mk_lane = [&](int kl, int w) {
    return mk_row(kl) + 128 * ((w + (kl & 1)) & 3) + 16 * ((li & 3) >> 1) + 8 * (li & 1);
  };
  const auto frag = [&](const char* S, int wbase, int i) {
    const int w = wbase / 64 + i / 4;
    return lds_tr_pair(S + mk_lane(kl1, w) + 32 * (i % 4), S + mk_lane(kl2, w) + 32 * (i % 4));
  };

  int claim = 0;  // lane 0 of wave 0: the own-XCD counter's value for the tile after the current one
  setup(L, cur);
  issue_all(0);
  issue_all(1);
  issue_all(2);
  issue_all(3);
  if (tid == 0) claim = __hip_atomic_fetch_add(queues + xcc, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();  // every wave has read next_tile
  for (;;) {
    floatx4 acc[8][8];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this tile's first loads (and any earlier stores) are done
    barrier();
    const int KTN2 = (KTN + 1) & ~1;
    if (!cur.cols) {
      for (int kt = 0; kt < KTN2; ++kt) {
        wait_vmcnt<16>();
        barrier();
        issue_all(kt + 4);
      }
    } else {
      Chunk fa[2][8], fb[2][8];
#pragma unroll
      for (int i = 0; i < 8; ++i) fa[0][i] = frag(smem, wm * C::WTM, i);
#pragma unroll
      for (int j = 0; j < 8; ++j) fb[0][j] = frag(smem + C::A_BYTES, wn * C::WTN, j);
      const auto step = [&](int kt, auto set) {
        constexpr int S = decltype(set)::value;
        const char* As = smem + ((kt + 1) & 3) * C::STAGE_BYTES;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const int m = i * 8 + j;
            if (m == 16) {
              wait_vmcnt<16>();  // K-tile kt + 1 has landed
              barrier();
            }
            mfma_bf16_agpr(acc[i][j], fb[S][j], fa[S][i]);
            if (m >= 16) {
              const int r = m - 16;
              if (r % 3 == 0) {
                const int t = r / 3;
                if (t == 0) fa[S ^ 1][0] = frag(As, wm * C::WTM, 0);
                else if (t <= 8) fb[S ^ 1][t - 1] = frag(As + C::A_BYTES, wn * C::WTN, t - 1);
                else fa[S ^ 1][t - 8] = frag(As, wm * C::WTM, t - 8);
              }
              if (r % 6 == 2) load_one(kt + 4, r / 6);
            }
          }
        }
      };
      for (int kt = 0; kt < KTN2; kt += 2) {
        step(kt, std::integral_constant<int, 0>{});
        step(kt + 1, std::integral_constant<int, 1>{});
      }
    }
    wait_vmcnt<0>();  // the zero-filling loads past the last K-tile have landed
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
    if (tid == 0) {
      const int Lc = wg_tile_of(claim, xcc, n_tiles);
      next_tile = Lc >= 0 ? Lc : wg_steal(queues, xcc, n_tiles);
    }
    __syncthreads();  // every wave is done with the ring; next_tile is visible
    const int Ln = next_tile;
    const WgTile done = cur;
    if (Ln >= 0) {
      setup(Ln, cur);
      issue_all(0);
      issue_all(1);
      issue_all(2);
      issue_all(3);
      if (tid == 0) claim = __hip_atomic_fetch_add(queues + xcc, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    // the finished tile, through this wave's staging area past the ring
    if (done.cols) {
      constexpr int CPRW = C::WTN / 8;
#pragma unroll
      for (int part = 0; part < 8; ++part) {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const floatx4 v = acc[part][j];
          uint2 pk;
          pk.x = pack_bf16x2(v[0], v[1]);
          pk.y = pack_bf16x2(v[2], v[3]);
          *reinterpret_cast<uint2*>(stg + (li * P16 + 16 * j + 4 * q) * 2) = pk;
        }
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int it = 0; it < STG_ROWS * CPRW / 64; ++it) {
          const int qq = lane + 64 * it, rr = qq / CPRW, cc = (qq % CPRW) * 8;
          const int m = done.m0 + wm * C::WTM + part * STG_ROWS + rr;
          const Chunk v = *reinterpret_cast<const Chunk*>(stg + (rr * P16 + cc) * 2);
          const int col = done.n0 + wn * C::WTN + cc;
          if (KIND == WG_DOWN) {
            st_chunk_nt((char*)p.out + (((size_t)done.g * d + m) * f + col) * ES, v);
          } else {
            char* o = (m < f) ? (char*)p.out + (((size_t)done.g * f + m) * d + col) * ES
                              : (char*)p.out2 + (((size_t)done.g * f + (m - f)) * d + col) * ES;
            st_chunk_nt(o, v);
          }
        }
        __builtin_amdgcn_wave_barrier();
      }
    }
    if (Ln < 0) return;
  }
}

// Two independent contractions in one launch: workgroups [0, grid_a) take tiles of KA (the longer
// K loops, so they start first), the next ones tiles of KB. The CUs that KA's tile grid leaves idle
// work through KB meanwhile, instead of idling until the next launch.
// KB's last `dyn` tiles are claimed at run time: each of the `dyn_wg` workgroups from `dyn_first` on takes a
// ticket (an agent-scope counter that starts at zero) and computes KB tile tiles_b - dyn + ticket, or nothing once
// the tickets run out. The hardware deals workgroups to the XCDs in turn, whatever their speed; with a share of
// the tiles left unassigned, the XCDs that run ahead take more of them and all finish together.
template <int BM, int BN, int BK, int KA, int KB, int STAGES, int WM, int WN>
__global__ __launch_bounds__(64 * WM * WN) __attribute__((amdgpu_waves_per_eu(
    Cfg2<BM, BN, BK, STAGES, WM, WN>::WAVES_PER_EU))) void gemm_bf16_pair_kernel(GemmArgs pa, GemmArgs pb,
                                                                                 int grid_a, int dyn_first,
                                                                                 int dyn, int tiles_b,
                                                                                 int* tickets) {
  extern __shared__ __align__(16) char smem[];
  __shared__ int ticket;
  const int bid = blockIdx.x;
  if (bid < grid_a) {
    gemm_tile<BM, BN, BK, KA, STAGES, WM, WN>(pa, bid, smem);
  } else if (dyn < 0) {  // persistent workgroups for KB (see wg_persistent)
    if constexpr (Cfg2<BM, BN, BK, STAGES, WM, WN>::PIPE && STAGES == 4 && (KB == WG_DOWN || KB == WG_GU))
      wg_persistent<KB>(pb, smem, tickets, tiles_b);
  } else if (bid < dyn_first) {
    gemm_tile<BM, BN, BK, KB, STAGES, WM, WN>(pb, bid - grid_a, smem);
  } else {
    if (threadIdx.x == 0) ticket = __hip_atomic_fetch_add(tickets, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    const int t = ticket;
    if (t < dyn) gemm_tile<BM, BN, BK, KB, STAGES, WM, WN>(pb, tiles_b - dyn + t, smem);
  }
}

// Zeroes the tickets of the paired launches that follow on the stream.
__global__ void zero_tickets_kernel(int* p, int n) {
  if ((int)threadIdx.x < n) p[threadIdx.x] = 0;
}

// ------------------------------------------------------------------------- host side

static int device_cus();
// Ticket-claimed tiles (see gemm_bf16_pair_kernel): 1 by default, PCMOE_DYN=0 keeps every tile on the workgroup its
// index implies, PCMOE_DYN=2 claims some tiles by ticket at any size.
static int dynamic_tiles() {
  static const int mode = [] {
    const char* env = getenv("PCMOE_DYN");
    return env && (env[0] == '0' || env[0] == '2') ? env[0] - '0' : 1;
  }();
  return mode;
}
template <int BM, int BN, int BK, int KIND, int STAGES, int WM, int WN>
static hipError_t run2(const GemmArgs& a, long tiles, hipStream_t s, const char* name) {
  using C = Cfg2<BM, BN, BK, STAGES, WM, WN>;
  static_assert(C::LDS <= 160 * 1024, "LDS budget of one CU");
  auto kern = gemm_bf16_kernel<BM, BN, BK, KIND, STAGES, WM, WN>;
  static std::atomic<uint64_t> lds_set{0};
  if (hipError_t e = lds_limit_once((const void*)kern, C::LDS, lds_set); e != hipSuccess) return e;
  const int grid = (int)((tiles + 7) / 8 * 8);
  if (grid <= 0) return hipSuccess;
  // with a.tickets, the last eighth of the grid's workgroup indices is claimed by ticket (as in the paired launches)
  int dyn = 0;
  if (a.tickets && dynamic_tiles() == 2) dyn = std::min(grid, std::max(grid / 64 * 8, 8));
  else if (a.tickets && grid >= 8 * device_cus()) dyn = grid / 64 * 8;
  const int dyn_first = grid - dyn, dyn_wg = dyn > 0 ? dyn + 256 : 0;
  KernelTimer kt(name, s);
  hipLaunchKernelGGL(kern, dim3(dyn_first + dyn_wg), dim3(C::NT), C::LDS, s, a, dyn_first, dyn);
  return hipGetLastError();
}

// Tile shapes (BM x BN, LDS stages, wavefronts) instantiated for every contraction. The default is
// 256 x 256 with 16 wavefronts (one workgroup per CU, four wavefronts per SIMD); 4-wavefront 128 x 128
// tiles run two workgroups per CU. The other shapes are selectable for measurement (PCMOE_GEMM_TILES).
// 192-row tiles (K-contiguous A only: the row-ragged contractions) serve a contraction whose 256-row grid is
// one partial round of the chip.
enum TileShape { T128x128s2 = 0, T256x128w8, T128x256w8, T256x256w8, T256x256k32, T256x128k32, T128x128k32,
                 T256x256w16, T256x256w16k32s4, T256x256w16k32s3, T192x256w8, T256x256w4, N_SHAPES };
static const int kShapeBM[N_SHAPES] = {128, 256, 128, 256, 256, 256, 128, 256, 256, 256, 192, 256};
static const int kShapeBN[N_SHAPES] = {128, 128, 256, 256, 256, 128, 128, 256, 256, 256, 256, 256};
static const char* kShapeName[N_SHAPES] = {"128x128s2", "256x128w8", "128x256w8", "256x256w8", "256x256k32",
                                           "256x128k32", "128x128k32", "256x256w16", "256x256w16k32s4",
                                           "256x256w16k32s3", "192x256w8", "256x256w4"};

static const char* kKindName[6] = {"gemm_fwd_gate_up", "gemm_fwd_down", "gemm_bwd_dh", "gemm_bwd_dx",
                                   "gemm_wgrad_down", "gemm_wgrad_gate_up"};

// PCMOE_PERSIST=0 keeps the pipelined weight gradients on ticket-claimed tails instead of persistent workgroups.
static bool persistent_wgrad() {
  static const bool on = [] {
    const char* env = getenv("PCMOE_PERSIST");
    return !(env && env[0] == '0');
  }();
  return on;
}
template <int BM, int BN, int BK, int KA, int KB, int STAGES, int WM, int WN>
static hipError_t run_pair2(const GemmArgs& a, long tiles_a, const GemmArgs& b, long tiles_b, int* tickets,
                            hipStream_t s, const char* name) {
  using C = Cfg2<BM, BN, BK, STAGES, WM, WN>;
  // the persistent weight-gradient loop stages its epilogue past the operand ring
  constexpr bool PERSIST = C::PIPE && STAGES == 4 && (KB == WG_DOWN || KB == WG_GU);
  constexpr int LDS = PERSIST ? (C::LDS > WG_LDS ? C::LDS : WG_LDS) : C::LDS;
  static_assert(LDS <= 160 * 1024, "LDS budget of one CU");
  auto kern = gemm_bf16_pair_kernel<BM, BN, BK, KA, KB, STAGES, WM, WN>;
  static std::atomic<uint64_t> lds_set{0};
  if (hipError_t e = lds_limit_once((const void*)kern, LDS, lds_set); e != hipSuccess) return e;
  // grid_a a multiple of 8 keeps each workgroup of the second contraction on the XCD its index implies
  const int grid_a = (int)((tiles_a + 7) / 8 * 8);
  // KB's last eighth of tiles (a multiple of 8) goes to ticket-taking workgroups, 32 more per XCD than tiles, when
  // KB fills at least 8 rounds of the chip (the extra workgroups cost a few microseconds at the launch's end);
  // PCMOE_DYN=2 takes at least 8 tiles (all of them below 8) this way at any size
  int dyn = 0;
  if (tickets && dynamic_tiles() == 2) dyn = (int)std::min<long>(tiles_b, std::max<long>(tiles_b / 64 * 8, 8));
  else if (tickets && tiles_b >= 8L * device_cus()) dyn = (int)(tiles_b / 64 * 8);
  int dyn_wg = dyn > 0 ? dyn + 256 : 0;
  int dyn_first = grid_a + (int)tiles_b - dyn;
  // The pipelined tile's weight gradients run in persistent workgroups instead (one per CU; see wg_persistent)
  if constexpr (PERSIST) {
    if (dyn > 0 && persistent_wgrad()) {
      dyn = -1;
      dyn_first = grid_a;
      dyn_wg = device_cus();
    }
  }
  const int grid = dyn_first + dyn_wg;
  if (grid <= 0) return hipSuccess;
  KernelTimer kt(name, s);
  hipLaunchKernelGGL(kern, dim3(grid), dim3(C::NT), LDS, s, a, b, grid_a, dyn_first, dyn, (int)tiles_b, tickets);
  return hipGetLastError();
}

template <int KIND>
static hipError_t run_shape(int shape, const GemmArgs& a, long tiles, hipStream_t s) {
  switch (shape) {
    case T128x128s2: return run2<128, 128, 64, KIND, 2, 2, 2>(a, tiles, s, kKindName[KIND]);
    case T256x128w8: return run2<256, 128, 64, KIND, 2, 4, 2>(a, tiles, s, kKindName[KIND]);
    case T128x256w8: return run2<128, 256, 64, KIND, 2, 2, 4>(a, tiles, s, kKindName[KIND]);
    case T256x256k32: return run2<256, 256, 32, KIND, 4, 2, 4>(a, tiles, s, kKindName[KIND]);
    case T256x128k32: return run2<256, 128, 32, KIND, 4, 4, 2>(a, tiles, s, kKindName[KIND]);
    case T128x128k32: return run2<128, 128, 32, KIND, 3, 2, 2>(a, tiles, s, kKindName[KIND]);
    case T256x256w16: return run2<256, 256, 64, KIND, 2, 4, 4>(a, tiles, s, kKindName[KIND]);
    case T256x256w16k32s4: return run2<256, 256, 32, KIND, 4, 4, 4>(a, tiles, s, kKindName[KIND]);
    case T256x256w16k32s3: return run2<256, 256, 32, KIND, 3, 4, 4>(a, tiles, s, kKindName[KIND]);
    case T256x256w4: return run2<256, 256, 32, KIND, 4, 2, 2>(a, tiles, s, kKindName[KIND]);
    case T192x256w8:
      if constexpr (KindTraits<KIND>::a_kc) return run2<192, 256, 64, KIND, 2, 2, 4>(a, tiles, s, kKindName[KIND]);
      return hipErrorInvalidValue;  // not selected for K-major A (fit_shape)
    default: return run2<256, 256, 64, KIND, 2, 2, 4>(a, tiles, s, kKindName[KIND]);
  }
}

// Default shape per contraction; PCMOE_GEMM_TILES="<kind>=<shape>,..." overrides (kind 0..5 as in
// GemmKind, shape as in kShapeName), e.g. "0=256x256s2,5=128x256s3".
static long mtile_bound2(const moe_desc& d, int bm);
static int tile_shape(int kind, const moe_desc& d) {
  struct Overrides {  // parsed once (thread-safe static initialisation)
    int table[6] = {-1, -1, -1, -1, -1, -1};
    Overrides() {
      const char* p = getenv("PCMOE_GEMM_TILES");
      while (p && *p) {
        int k = *p - '0';
        if (k >= 0 && k < 6 && p[1] == '=') {
          for (int sh = 0; sh < N_SHAPES; ++sh)
            if (!strncmp(p + 2, kShapeName[sh], strlen(kShapeName[sh]))) table[k] = sh;
        }
        while (*p && *p != ',') ++p;
        if (*p == ',') ++p;
      }
    }
  };
  static const Overrides ov;
  if (ov.table[kind] >= 0) return ov.table[kind];
  // FWD_DOWN (N = d_model): when its 256x256 grid is one partial round of the chip, 192-row tiles still fit one
  // round and each costs about 3/4 of a 256-row tile. (The backward kinds run paired with a weight gradient,
  // which shares their shape.)
  if (kind == FWD_DOWN) {
    if (d.d_model % 256 == 0) {
      const long n = d.d_model / 256;
      if (mtile_bound2(d, 256) * n <= device_cus() && mtile_bound2(d, 192) * n <= device_cus()) return T192x256w8;
    }
    return T256x256w16;
  }
  // The pipelined 4-wavefront tile pays off on long K loops only: its prologue and epilogue (one wavefront per
  // SIMD, each storing four times the outputs of a 16-wavefront tile's wavefront) are amortised over K. Measured:
  // 1.6% faster per layer step at d_model = 4096 (the dX + dW_gate|up pair 3.4%), equal at d_model = 2048 with
  // 64 experts, 3% slower for a 16-expert shard at d_model = 2048 and 7% slower at d_model = 1024. With persistent
  // weight-gradient workgroups, the dX + dW_gate|up pair also gains where its dX grid fills 8 rounds of the chip
  // (d_model = 2048 with 64 experts: 6%), while the other kinds there stay faster on the 16-wavefront tile.
  if (d.d_model >= 4096) return T256x256w4;
  if ((kind == BWD_DX || kind == WG_GU) && d.d_model % 256 == 0 &&
      mtile_bound2(d, 256) * (d.d_model / 256) >= 8L * device_cus())
    return T256x256w4;
  return T256x256w16;
}

// Upper bound on the m-tiles of the row-ragged kinds (per-expert counts stay on the device).
static long mtile_bound2(const moe_desc& d, int bm) {
  long routed = ((long)d.T * d.top_k + (long)d.local_count * (bm - 1)) / bm;
  return routed + (long)d.n_shared * ((d.T + bm - 1) / bm);
}

static size_t plan_part(const moe_desc& d) { return align256((size_t)(d.local_count + d.n_shared + 1) * 4); }
static size_t plan_bytes(const moe_desc& d) { return 6 * plan_part(d); }
// saved = G|U [R, 2f], H [R, f], then the tile plan of the forward, which the backward reuses
static size_t saved_plan_offset(const moe_desc& d) {
  const size_t R = (size_t)rows_total(d), es = elem_bytes(d);
  return align256(R * 2 * d.d_ff * es) + align256(R * d.d_ff * es);
}
// ... and 256 bytes for the forward launches' tile tickets
size_t ffn_saved_bytes(const moe_desc& d) { return saved_plan_offset(d) + align256(plan_bytes(d)) + 256; }
size_t ffn_fwd_ws_bytes(const moe_desc&) { return 0; }
// dG|dU [R, 2f], then the tickets of the two paired launches (bf16)
size_t ffn_bwd_ws_bytes(const moe_desc& d) {
  const size_t R = (size_t)rows_total(d), es = elem_bytes(d);
  return align256(R * 2 * d.d_ff * es) + 256;
}

struct Plan {
  int32_t* pre128;
  int32_t* pre256;
  int32_t* order;
  int32_t* body256;  // 256-row m-tiles other than the tails
  int32_t* tail256;  // 256-row tail m-tiles (at most 128 rows)
  int32_t* pre192;
};

// The plan's arrays at `where`: m-tile prefixes for 128-, 192- and 256-row tiles, the heaviest-first group order,
// and for 256-row tiles the prefixes without the tails and of the tails.
static Plan plan_at(const moe_desc& d, void* where) {
  Plan pl;
  pl.pre128 = (int32_t*)where;
  pl.pre256 = (int32_t*)((char*)where + plan_part(d));
  pl.order = (int32_t*)((char*)where + 2 * plan_part(d));
  pl.body256 = (int32_t*)((char*)where + 3 * plan_part(d));
  pl.tail256 = (int32_t*)((char*)where + 4 * plan_part(d));
  pl.pre192 = (int32_t*)((char*)where + 5 * plan_part(d));
  return pl;
}
// (zero, nzero: counters the plan kernel also clears, for the launches that follow it)
static Plan plan(const moe_desc& d, const int32_t* offsets, void* where, hipStream_t s, int32_t* zero = nullptr,
                 int nzero = 0) {
  Plan pl = plan_at(d, where);
  KernelTimer kt("ffn_plan", s);
  hipLaunchKernelGGL(mtile_prefix_kernel, dim3(1), dim3(512), 0, s, offsets, d.local_count, d.n_shared, d.T, 128, 256,
                     192, pl.pre128, pl.pre256, pl.body256, pl.tail256, pl.pre192, pl.order, zero, nzero);
  return pl;
}

static GemmArgs args_for(const moe_desc& d, const int32_t* offsets) {
  GemmArgs a{};
  a.T = d.T; a.k = d.top_k; a.d = d.d_model; a.f = d.d_ff; a.Eloc = d.local_count; a.S = d.n_shared;
  a.rows_cap = d.T * d.top_k;
  a.offsets = offsets;
  return a;
}

// Compute units of the current device (queried once per device).
static int device_cus() {
  static std::atomic<int> cus[64];  // 0 = not queried yet
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  int c = cus[dev].load(std::memory_order_relaxed);
  if (c <= 0) {
    int n = 0;
    c = (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && n > 0) ? n : 256;
    cus[dev].store(c, std::memory_order_relaxed);
  }
  return c;
}

// Ragged-M contraction: n_cols output columns of the tile grid (FWD_GU: gate columns, two per pair).
// A shape must tile M exactly (d_model, d_ff are multiples of 128), else it falls back to 128-wide sides. Along N
// the 256 x 256 tile also takes a last n-tile of 128 columns (N an odd multiple of 128, e.g. d_ff = 1408): its
// upper two wave columns skip their MFMAs and stores. Other shapes need N to be a multiple of their width.
static int fit_shape(int sh, int M, int N) {
  int bm = kShapeBM[sh], bn = kShapeBN[sh];
  if (M > 0 && (M % bm || bm == 192)) bm = 128;  // weight gradients (K-major A) take no 192-row tiles
  if (N % bn && !((sh == T256x256w16 || sh == T256x256w4) && N % 128 == 0)) bn = 128;
  if (bm == kShapeBM[sh] && bn == kShapeBN[sh]) return sh;
  const bool k32 = sh == T256x256k32 || sh == T256x128k32 || sh == T128x128k32;
  if (sh == T256x256w16 || sh == T256x256w16k32s4 || sh == T256x256w16k32s3 || sh == T256x256w4)
    return T128x128s2;  // measured best when one side must drop to 128
  if (bm == 256 && bn == 128) return k32 ? T256x128k32 : T256x128w8;
  if (bm == 128 && bn == 256) return T128x256w8;
  return k32 ? T128x128k32 : T128x128s2;
}

// A contraction ready to launch: tile shape, arguments and the workgroups its grid needs.
struct Prep {
  int sh;
  GemmArgs a;
  long tiles;
};

// Column windows per tail tile of the down projection: 4 (PCMOE_TAIL_SPLIT=1, 2 or 4 overrides).
static int tail_split_windows() {
  static const int ts = [] {
    const char* env = getenv("PCMOE_TAIL_SPLIT");
    return env && (env[0] == '1' || env[0] == '2' || env[0] == '4') ? env[0] - '0' : 4;
  }();
  return ts;
}

// Ragged-M contraction with n_cols output columns in the tile grid (FWD_GU: gate and up columns). tails_last:
// split off the tails even when the grid is one round (a paired launch, where it shares the chip).
template <int KIND>
static Prep prep_ragged(const moe_desc& d, GemmArgs a, const Plan& pl, int n_cols, bool tails_last = false) {
  const int sh = fit_shape(tile_shape(KIND, d), 0, n_cols);
  const int bm = kShapeBM[sh], bn = kShapeBN[sh];
  a.n_tiles = (n_cols + bn - 1) / bn;  // FWD_GU: n_cols = 2f, each tile holds bn/2 gate and bn/2 up columns
  a.n_extent = n_cols;
  const long bound = mtile_bound2(d, bm) * a.n_tiles;
  // 256-row tiles in more than one round of the chip, or sharing it with another contraction: tails after the
  // others (see decode_tile), so that every XCD gets an even share of both; its share of each segment is rounded
  // up, at most 16 workgroups more
  const bool split = bm == 256 && (tails_last || bound > device_cus());
  a.mt_prefix = bm == 128 ? pl.pre128 : bm == 192 ? pl.pre192 : split ? pl.body256 : pl.pre256;
  a.mt_tail = split ? pl.tail256 : nullptr;
  // A down projection of a few rounds runs its tails (at most half a tile of rows each) in a last, partial round,
  // where each tail tile still loads its whole B panel and most CUs idle. Split into column windows (one per
  // workgroup, consecutive in the tail segment), the tails load a window's B rows each and spread over those CUs;
  // the decode takes fewer windows per tile when those of all the tails would not fit the CUs. Each group has at
  // most one tail m-tile: the windows add at most (tail_split - 1) * G * n_tiles workgroups.
  long extra = 0;
  if (KIND == FWD_DOWN && split && sh == T256x256w16 && bound <= 8L * device_cus()) {
    a.tail_split = tail_split_windows();
    a.tail_cus = device_cus();
    extra = (long)(a.tail_split - 1) * (d.local_count + d.n_shared) * a.n_tiles;
  }
  return Prep{sh, a, bound + (split ? 16 : 0) + extra};
}
// Weight gradient: an M x N output per group, K = the group's rows.
template <int KIND>
static Prep prep_wgrad(const moe_desc& d, GemmArgs a, const Plan& pl, int M, int N) {
  const int sh = fit_shape(tile_shape(KIND, d), M, N);
  a.order = pl.order;
  // dW_gate|dW_up takes its groups round-robin: it shares its launch with dX, whose tiles read the same dG|dU
  // rows, and every group's rows then get pulled into the caches early, not only the heaviest groups'.
  // PCMOE_WGRR=<bit mask of kinds> overrides.
  static const int wgrr = [] {
    const char* e = getenv("PCMOE_WGRR");
    return e ? atoi(e) : -1;
  }();
  a.wg_interleave = wgrr >= 0 ? (wgrr >> KIND) & 1 : (KIND == WG_GU ? 1 : 0);
  a.m_tiles = M / kShapeBM[sh];
  a.n_tiles = (N + kShapeBN[sh] - 1) / kShapeBN[sh];
  a.n_extent = N;
  return Prep{sh, a, (long)(d.local_count + d.n_shared) * a.m_tiles * a.n_tiles};
}
template <int KIND>
static hipError_t run(const Prep& p, hipStream_t s) {
  return run_shape<KIND>(p.sh, p.a, p.tiles, s);
}


// PCMOE_PAIR=0 launches the paired contractions one after the other instead.
static bool pair_enabled() {
  static const bool on = [] {
    const char* env = getenv("PCMOE_PAIR");
    return !(env && env[0] == '0');
  }();
  return on;
}

// Whether run_pair below launches A and B together with B's last tiles claimed at run time (by ticket or by
// persistent workgroups), that is whether it reads the tile counters it is given: the condition run_pair2 applies.
static bool pair_claims(const Prep& A, const Prep& B) {
  if (!pair_enabled() || A.sh != B.sh) return false;
  if (A.sh != T256x256w16 && A.sh != T256x256w4 && A.sh != T128x128s2) return false;  // no paired kernel
  return dynamic_tiles() == 2 || B.tiles >= 8L * device_cus();
}

// Independent contractions A and B (no operand of one is written by the other) in one launch when
// they share a tile shape; A's workgroups come first.
template <int KA, int KB>
static hipError_t run_pair(const Prep& A, const Prep& B, int* tickets, hipStream_t s, const char* name) {
  if (A.sh == B.sh && pair_enabled()) {
    switch (A.sh) {
      case T256x256w16:
        return run_pair2<256, 256, 64, KA, KB, 2, 4, 4>(A.a, A.tiles, B.a, B.tiles, tickets, s, name);
      case T256x256w4:
        return run_pair2<256, 256, 32, KA, KB, 4, 2, 2>(A.a, A.tiles, B.a, B.tiles, tickets, s, name);
      case T128x128s2:
        return run_pair2<128, 128, 64, KA, KB, 2, 2, 2>(A.a, A.tiles, B.a, B.tiles, tickets, s, name);
      default: break;
    }
  }
  hipError_t e = run<KA>(A, s);
  if (e != hipSuccess) return e;
  return run<KB>(B, s);
}

hipError_t launch_ffn_fwd(const moe_desc& d, const void* x, const void* xp, const int32_t* offsets, const void* wg,
                          const void* wu, const void* wd, void* yp, void* saved, void*, hipStream_t s) {
  // the gate/up and down-projection tile counters (after the plan in the saved buffer), cleared by the plan kernel
  int* tickets = (int*)((char*)saved + saved_plan_offset(d) + align256(plan_bytes(d)));
  Plan pl = plan(d, offsets, (char*)saved + saved_plan_offset(d), s, tickets, 2);
  if (d.dtype != MOE_BF16) return ffn_fwd_f32(d, x, xp, offsets, wg, wu, wd, yp, saved, pl.pre128, s);
  const size_t R = (size_t)rows_total(d);
  GemmArgs a = args_for(d, offsets);
  a.x = x; a.xp = xp; a.wg = wg; a.wu = wu; a.wd = wd;
  a.gu = saved;
  a.h = (char*)saved + align256(R * 2 * d.d_ff * 2);
  a.out = yp;
  hipError_t e;
  GemmArgs a_gu = a, a_down = a;
  if (dynamic_tiles()) {
    a_gu.tickets = tickets;
    a_down.tickets = tickets + 1;
  }
  if ((e = run<FWD_GU>(prep_ragged<FWD_GU>(d, a_gu, pl, 2 * d.d_ff), s)) != hipSuccess) return e;
  return run<FWD_DOWN>(prep_ragged<FWD_DOWN>(d, a_down, pl, d.d_model), s);
}

hipError_t launch_ffn_bwd(const moe_desc& d, const void* x, const void* xp, const void* dy, const void* dyp,
                          const int32_t* offsets, const void* wg, const void* wu, const void* wd, const void* saved,
                          void* dxp, void* dwg, void* dwu, void* dwd, void* ws, hipStream_t s) {
  const size_t R = (size_t)rows_total(d), es = elem_bytes(d);
  void* dgu = ws;
  (void)es;
  Plan pl = plan_at(d, (char*)saved + saved_plan_offset(d));  // written by the forward for the same offsets
  if (d.dtype != MOE_BF16)
    return ffn_bwd_f32(d, x, xp, dy, dyp, offsets, wg, wu, wd, saved, dxp, dwg, dwu, dwd, dgu, pl.pre128, s);
  GemmArgs a = args_for(d, offsets);
  a.x = x; a.xp = xp; a.dy = dy; a.dyp = dyp; a.wg = wg; a.wu = wu; a.wd = wd;
  a.gu = (void*)saved;
  a.h = (char*)saved + align256(R * 2 * d.d_ff * 2);
  a.dgu = dgu;
  // dG|dU (BWD_DH) and dW_down (WG_DOWN) read only forward results and dY; dX (BWD_DX) and
  // dW_gate|dW_up (WG_GU) both read dG|dU.
  GemmArgs a_wd = a, a_wgu = a, a_dx = a;
  a_wd.out = dwd;
  a_wgu.out = dwg;
  a_wgu.out2 = dwu;
  a_dx.out = dxp;
  int* tickets = (int*)((char*)ws + align256(R * 2 * d.d_ff * es));
  const Prep dh = prep_ragged<BWD_DH>(d, a, pl, d.d_ff), wd_ = prep_wgrad<WG_DOWN>(d, a_wd, pl, d.d_model, d.d_ff);
  const Prep dx = prep_ragged<BWD_DX>(d, a_dx, pl, d.d_model, pair_enabled()),
             wgu = prep_wgrad<WG_GU>(d, a_wgu, pl, 2 * d.d_ff, d.d_model);
  // the counters are read only by paired launches that claim tiles at run time: cleared (one launch) only then
  if (dynamic_tiles() && (pair_claims(dh, wd_) || pair_claims(dx, wgu))) {
    hipLaunchKernelGGL(zero_tickets_kernel, dim3(1), dim3(64), 0, s, tickets, 16);
    if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
  }
  hipError_t e = run_pair<BWD_DH, WG_DOWN>(dh, wd_, dynamic_tiles() ? tickets : nullptr, s, "gemm_bwd_dh+wgrad_down");
  if (e != hipSuccess) return e;
  return run_pair<BWD_DX, WG_GU>(dx, wgu, dynamic_tiles() ? tickets + 8 : nullptr, s, "gemm_bwd_dx+wgrad_gate_up");
}

}  // namespace pcmoe
