// Expert passes of Alg. 6 (ForwardExpert / BackwardExpert) as grouped GEMMs — fp32 storage path
// (v_mfma_f32_16x16x4_f32, register-staged double buffer). The bf16 path is grouped_gemm_bf16.hip.
//
// One kernel template covers the six contractions of a SwiGLU expert:
//   FWD_GU   [G|U] = h W_{gate|up}^T, epilogue H = silu(G) * U    (M = rows, N = 2f, K = d)
//   FWD_DOWN O = H W_down^T                                       (M = rows, N = d,  K = f)
//   BWD_DH   dH = dO W_down, epilogue dG, dU (SwiGLU adjoint)      (M = rows, N = f,  K = d)
//   BWD_DX   dh = [dG|dU] [W_gate;W_up]                            (M = rows, N = d,  K = 2f)
//   WG_DOWN  dW_down = dO^T H                                      (M = d,  N = f,  K = rows)
//   WG_GU    [dW_gate;dW_up] = [dG|dU]^T h                         (M = 2f, N = d,  K = rows)
// Groups are the hosted routed experts (rows from the dispatch offsets, read on the device) and
// the shared experts (all T tokens). Tiles: BM x BN per workgroup of 2x2 wavefronts, K staged in
// LDS 128 bytes per row (64 bf16 / 32 fp32) with a 16-byte-chunk XOR swizzle, double-buffered,
// fp32 accumulation in MFMA registers (bf16: v_mfma_f32_16x16x32_bf16, fp32: v_mfma_f32_16x16x4_f32).
// Operands whose K dimension is not contiguous in memory are transposed in registers on their
// way to LDS (8x8 blocks of bf16 / 4x4 of fp32), so the MFMA side always reads K-contiguous rows.
// Epilogues stage the fp32 tile through LDS and write 16-byte chunks.
#include "grouped_gemm.h"

namespace pcmoe {

__device__ __forceinline__ int swz(int r) { return ((r >> 1) ^ (r >> 4)) & 7; }
__device__ __forceinline__ int lds_off(int r, int c) { return r * 128 + ((c ^ swz(r)) << 4); }

template <typename T> struct Mfma;
template <> struct Mfma<bf16> {
  static __device__ __forceinline__ void run(floatx4& acc, const Chunk& a, const Chunk& b) {
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), acc,
                                                  0, 0, 0);
  }
};
template <> struct Mfma<float> {
  static __device__ __forceinline__ void run(floatx4& acc, const Chunk& a, const Chunk& b) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w[i]), __uint_as_float(b.w[i]), acc, 0, 0, 0);
  }
};

// Transpose an EPC x EPC block held as EPC chunks (row i = chunk i) so that out[m] holds column m.
__device__ __forceinline__ void transpose_block(const Chunk* in, Chunk* out, bf16) {
#pragma unroll
  for (int m = 0; m < 8; ++m) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t lo = in[2 * j].w[m >> 1], hi = in[2 * j + 1].w[m >> 1];
      out[m].w[j] = (m & 1) ? ((lo >> 16) | (hi & 0xffff0000u)) : ((lo & 0xffffu) | (hi << 16));
    }
  }
}
__device__ __forceinline__ void transpose_block(const Chunk* in, Chunk* out, float) {
#pragma unroll
  for (int m = 0; m < 4; ++m)
#pragma unroll
    for (int j = 0; j < 4; ++j) out[m].w[j] = in[j].w[m];
}

template <typename T, int BM, int BN, int WM, int WN>
struct TileCfg {
  static constexpr int NT = 64 * WM * WN;
  static constexpr int EPCN = EPC<T>::value;
  static constexpr int BK = 8 * EPCN;              // elements per 128-byte LDS row
  static constexpr int WTM = BM / WM, WTN = BN / WN;
  static constexpr int FM = WTM / 16, FN = WTN / 16;
  static constexpr int CP = BN + 16;               // fp32 pitch of the epilogue tile
  static constexpr int LDS_MAIN = 2 * (BM + BN) * 128;
  static constexpr int LDS_EPI = BM * CP * 4;
  static constexpr int LDS = LDS_MAIN > LDS_EPI ? LDS_MAIN : LDS_EPI;
};

// Loader of a K-contiguous operand tile: R rows x 8 chunks, NT threads.
template <int R, int NT>
struct KcLoader {
  static constexpr int N = (R * 8 + NT - 1) / NT;
  const char* src[N];
  int off[N];
  Chunk reg[N];
  __device__ __forceinline__ void load(int kbyte) {
#pragma unroll
    for (int i = 0; i < N; ++i) reg[i] = src[i] ? ld_chunk(src[i] + kbyte) : zero_chunk();
  }
  __device__ __forceinline__ void store(char* lds) {
#pragma unroll
    for (int i = 0; i < N; ++i)
      if (off[i] >= 0) st_chunk(lds + off[i], reg[i]);
  }
};

// Loader of an MN-contiguous operand tile (K rows in memory, R contiguous columns): EPC x EPC
// blocks, transposed in registers.
template <typename T, int R, int NT>
struct McLoader {
  static constexpr int E = EPC<T>::value;
  static constexpr int NBLK = 8 * (R / E);
  static constexpr int N = (NBLK + NT - 1) / NT;
  const char* src[N];   // column base of the block (row 0 of the tile), or null
  int kb[N];            // k-block (chunk index in LDS)
  int mb[N];            // mn-block
  Chunk reg[N][E];
  __device__ __forceinline__ void load(ptrdiff_t shift, int ld_bytes, int krow0, int kvalid) {
    // shift: byte offset added to src (selects the K-tile's source half); krow0: first K row
#pragma unroll
    for (int i = 0; i < N; ++i) {
#pragma unroll
      for (int r = 0; r < E; ++r) {
        const int kr = krow0 + kb[i] * E + r;
        reg[i][r] = (src[i] && kr < kvalid) ? ld_chunk(src[i] + shift + (size_t)kr * ld_bytes)
                                            : zero_chunk();
      }
    }
  }
  __device__ __forceinline__ void store(char* lds) {
#pragma unroll
    for (int i = 0; i < N; ++i) {
      if (kb[i] < 0) continue;
      Chunk tr[E];
      transpose_block(reg[i], tr, T());
      const int par = mb[i] & 1;
#pragma unroll
      for (int r = 0; r < E; ++r) {
        const int rr = r ^ par;  // alternate the row order of odd blocks: spreads LDS banks
        Chunk v;
#pragma unroll
        for (int q = 0; q < 4; ++q) v.w[q] = par ? tr[r ^ 1].w[q] : tr[r].w[q];
        st_chunk(lds + lds_off(mb[i] * E + rr, kb[i]), v);
      }
    }
  }
};

template <typename T, int BM, int BN, int WM, int WN, int KIND>
__global__ __launch_bounds__(64 * WM * WN) void grouped_gemm_kernel(GemmArgs p) {
  using C = TileCfg<T, BM, BN, WM, WN>;
  using KT = KindTraits<KIND>;
  constexpr int NT = C::NT, E = C::EPCN, BK = C::BK;
  extern __shared__ __align__(16) char smem[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;

  // ---------------------------------------------------------------- tile decode
  TileIdx ti;
  if (!decode_tile<KT::ragged_m>(p, blockIdx.x, ti)) return;
  const int g = ti.g, mt = ti.mt, nt = ti.nt;

  const bool routed = g < p.Eloc;
  const int row0 = ti.row0;                                          // first row of the group in its source
  const int rows = ti.rows;                                          // rows of the group
  const size_t rs = routed ? (size_t)row0 : (size_t)p.rows_cap + (size_t)(g - p.Eloc) * p.T;  // row-space base
  const int d = p.d, f = p.f;
  const size_t es = sizeof(T);

  const int m0 = mt * BM, n0 = nt * BN;
  int K;
  if (KIND == FWD_GU || KIND == BWD_DH) K = d;
  else if (KIND == FWD_DOWN) K = f;
  else if (KIND == BWD_DX) K = 2 * f;
  else K = rows;

  // ------------------------------------------------------------- operand setup
  KcLoader<BM, NT> akc;
  KcLoader<BN, NT> bkc;
  McLoader<T, BM, NT> amc;
  McLoader<T, BN, NT> bmc;
  int a_ld = 0, b_ld = 0;          // bytes
  ptrdiff_t b_half_shift = 0;      // BWD_DX: added to W_gate addresses for K rows >= f (W_up)

  if (KT::a_kc) {
    const char* abase;
    if (KIND == FWD_GU) { abase = routed ? (const char*)p.xp + rs * d * es : (const char*)p.x; a_ld = d * es; }
    else if (KIND == FWD_DOWN) { abase = (const char*)p.h + rs * f * es; a_ld = f * es; }
    else if (KIND == BWD_DH) { abase = routed ? (const char*)p.dyp + rs * d * es : (const char*)p.dy; a_ld = d * es; }
    else { abase = (const char*)p.dgu + rs * 2 * f * es; a_ld = 2 * f * es; }
#pragma unroll
    for (int i = 0; i < KcLoader<BM, NT>::N; ++i) {
      const int q = tid + i * NT;
      const int r = q >> 3, c = q & 7;
      const bool in_tile = r < BM;
      akc.off[i] = in_tile ? lds_off(r, c) : -1;
      akc.src[i] = (in_tile && m0 + r < rows) ? abase + (size_t)(m0 + r) * a_ld + c * 16 : nullptr;
    }
  } else {
    const char* abase;  // [K rows][M cols] with M contiguous
    if (KIND == WG_DOWN) { abase = routed ? (const char*)p.dyp + rs * d * es : (const char*)p.dy; a_ld = d * es; }
    else { abase = (const char*)p.dgu + rs * 2 * f * es; a_ld = 2 * f * es; }
#pragma unroll
    for (int i = 0; i < McLoader<T, BM, NT>::N; ++i) {
      const int blk = tid + i * NT;
      const bool ok = blk < McLoader<T, BM, NT>::NBLK;
      const int nmb = BM / E;
      amc.kb[i] = ok ? blk / nmb : -1;
      amc.mb[i] = ok ? blk % nmb : 0;
      amc.src[i] = ok ? abase + (size_t)(m0 + amc.mb[i] * E) * es : nullptr;
    }
  }
  if (KT::b_kc) {
#pragma unroll
    for (int i = 0; i < KcLoader<BN, NT>::N; ++i) {
      const int q = tid + i * NT;
      const int r = q >> 3, c = q & 7;
      const bool in_tile = r < BN;
      bkc.off[i] = in_tile ? lds_off(r, c) : -1;
      const char* src = nullptr;
      if (in_tile) {
        if (KIND == FWD_GU) {
          // LDS row r: wave column r / WTN; its first half are gate rows, the second half up rows
          const int wcol = r / C::WTN, within = r % C::WTN, half = C::WTN / 2;
          const int frow = nt * (BN / 2) + wcol * half + (within % half);
          const char* wsrc = (within < half) ? (const char*)p.wg : (const char*)p.wu;
          src = wsrc + ((size_t)g * f * d + (size_t)frow * d) * es + c * 16;
          b_ld = d * es;
        } else {  // FWD_DOWN: W_down[g] rows = output columns, K = f contiguous
          src = (const char*)p.wd + ((size_t)g * d * f + (size_t)(n0 + r) * f) * es + c * 16;
          b_ld = f * es;
        }
      }
      bkc.src[i] = src;
    }
  } else {
    const char* bbase;  // [K rows][N cols] with N contiguous, column n0
    if (KIND == BWD_DH) { bbase = (const char*)p.wd + (size_t)g * d * f * es; b_ld = f * es; }
    else if (KIND == BWD_DX) {
      bbase = (const char*)p.wg + (size_t)g * f * d * es;
      b_ld = d * es;
      b_half_shift = ((const char*)p.wu - (const char*)p.wg) - (ptrdiff_t)f * d * es;
    } else if (KIND == WG_DOWN) { bbase = (const char*)p.h + rs * f * es; b_ld = f * es; }
    else { bbase = routed ? (const char*)p.xp + rs * d * es : (const char*)p.x; b_ld = d * es; }
#pragma unroll
    for (int i = 0; i < McLoader<T, BN, NT>::N; ++i) {
      // B blocks start at the other half of the workgroup when A also needs the transposing loader
      const int tb = KT::a_kc ? tid : (tid + NT / 2) % NT;
      const int blk = tb + i * NT;
      const bool ok = blk < McLoader<T, BN, NT>::NBLK;
      const int nmb = BN / E;
      bmc.kb[i] = ok ? blk / nmb : -1;
      bmc.mb[i] = ok ? blk % nmb : 0;
      bmc.src[i] = ok ? bbase + (size_t)(n0 + bmc.mb[i] * E) * es : nullptr;
    }
  }

  // ---------------------------------------------------------------- main loop
  floatx4 acc[C::FM][C::FN];
#pragma unroll
  for (int i = 0; i < C::FM; ++i)
#pragma unroll
    for (int j = 0; j < C::FN; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  const int KT_N = (K + BK - 1) / BK;
  auto load_tile = [&](int kt) {
    const int k0 = kt * BK;
    if (KT::a_kc) akc.load(k0 * es);
    else amc.load(0, a_ld, k0, K);
    if (KT::b_kc) bkc.load(k0 * es);
    else bmc.load((KIND == BWD_DX && k0 >= f) ? b_half_shift : 0, b_ld, k0, K);
  };
  auto store_tile = [&](int buf) {
    char* As = smem + buf * (BM + BN) * 128;
    char* Bs = As + BM * 128;
    if (KT::a_kc) akc.store(As);
    else amc.store(As);
    if (KT::b_kc) bkc.store(Bs);
    else bmc.store(Bs);
  };

  if (KT_N > 0) {
    load_tile(0);
    store_tile(0);
  }
  __syncthreads();
  const int frow = lane & 15, fchunk = lane >> 4;
  for (int kt = 0; kt < KT_N; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < KT_N) load_tile(kt + 1);
    const char* As = smem + buf * (BM + BN) * 128;
    const char* Bs = As + BM * 128;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      Chunk a[C::FM], b[C::FN];
#pragma unroll
      for (int i = 0; i < C::FM; ++i) a[i] = ld_chunk(As + lds_off(wm * C::WTM + 16 * i + frow, 4 * kk + fchunk));
#pragma unroll
      for (int j = 0; j < C::FN; ++j) b[j] = ld_chunk(Bs + lds_off(wn * C::WTN + 16 * j + frow, 4 * kk + fchunk));
#pragma unroll
      for (int i = 0; i < C::FM; ++i)
#pragma unroll
        for (int j = 0; j < C::FN; ++j) Mfma<T>::run(acc[i][j], a[i], b[j]);
    }
    if (kt + 1 < KT_N) store_tile(buf ^ 1);
    __syncthreads();
  }

  // ---------------------------------------------------------------- epilogue
  float* Cs = reinterpret_cast<float*>(smem);
#pragma unroll
  for (int i = 0; i < C::FM; ++i) {
#pragma unroll
    for (int j = 0; j < C::FN; ++j) {
      int col;
      if (KIND == FWD_GU) {
        const int half = C::FN / 2;
        col = (j < half) ? wn * (C::WTN / 2) + 16 * j + frow
                         : BN / 2 + wn * (C::WTN / 2) + 16 * (j - half) + frow;
      } else {
        col = wn * C::WTN + 16 * j + frow;
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) Cs[(wm * C::WTM + 16 * i + 4 * fchunk + r) * C::CP + col] = acc[i][j][r];
    }
  }
  __syncthreads();

  constexpr int OUT_COLS = (KIND == FWD_GU) ? BN / 2 : BN;
  constexpr int CPR = OUT_COLS / E;  // output chunks per tile row
  for (int q = tid; q < BM * CPR; q += NT) {
    const int r = q / CPR, c = q % CPR;
    const int m = m0 + r;
    if (KT::ragged_m && m >= rows) continue;
    float v[E];
#pragma unroll
    for (int e = 0; e < E; ++e) v[e] = Cs[r * C::CP + c * E + e];
    if (KIND == FWD_GU) {
      float u[E], hv[E];
#pragma unroll
      for (int e = 0; e < E; ++e) {
        u[e] = Cs[r * C::CP + BN / 2 + c * E + e];
        const float sg = 1.f / (1.f + __expf(-v[e]));
        hv[e] = v[e] * sg * u[e];
      }
      const int col = nt * (BN / 2) + c * E;
      char* gu = (char*)p.gu + ((rs + m) * 2 * f + col) * es;
      st_chunk(gu, f_to_chunk<T>(v));
      st_chunk(gu + (size_t)f * es, f_to_chunk<T>(u));
      st_chunk((char*)p.h + ((rs + m) * f + col) * es, f_to_chunk<T>(hv));
    } else if (KIND == FWD_DOWN || KIND == BWD_DX) {
      st_chunk((char*)p.out + ((rs + m) * d + n0 + c * E) * es, f_to_chunk<T>(v));
    } else if (KIND == BWD_DH) {
      const int col = n0 + c * E;
      const char* gu = (const char*)p.gu + ((rs + m) * 2 * f + col) * es;
      float gv[E], uv[E], dg[E], du[E];
      chunk_to_f<T>(ld_chunk(gu), gv);
      chunk_to_f<T>(ld_chunk(gu + (size_t)f * es), uv);
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const float sg = 1.f / (1.f + __expf(-gv[e]));
        du[e] = v[e] * gv[e] * sg;
        dg[e] = v[e] * uv[e] * sg * (1.f + gv[e] * (1.f - sg));
      }
      char* o = (char*)p.dgu + ((rs + m) * 2 * f + col) * es;
      st_chunk(o, f_to_chunk<T>(dg));
      st_chunk(o + (size_t)f * es, f_to_chunk<T>(du));
    } else if (KIND == WG_DOWN) {
      st_chunk((char*)p.out + (((size_t)g * d + m) * f + n0 + c * E) * es, f_to_chunk<T>(v));
    } else {  // WG_GU
      char* o = (m < f) ? (char*)p.out + (((size_t)g * f + m) * d + n0 + c * E) * es
                        : (char*)p.out2 + (((size_t)g * f + (m - f)) * d + n0 + c * E) * es;
      st_chunk(o, f_to_chunk<T>(v));
    }
  }
}

// m-tile prefixes over groups for two tile heights: pre[g] = sum_{g' < g} ceil(rows_g' / bm); and
// the groups ordered by decreasing row count (ties by index).
__global__ __launch_bounds__(512) void mtile_prefix_kernel(const int32_t* __restrict__ offsets, int Eloc, int S,
                                                           int Tn, int bm0, int bm1, int bm2,
                                                           int32_t* __restrict__ pre0, int32_t* __restrict__ pre1,
                                                           int32_t* __restrict__ body1, int32_t* __restrict__ tail1,
                                                           int32_t* __restrict__ pre2, int32_t* __restrict__ order,
                                                           int32_t* __restrict__ zero, int nzero) {
  __shared__ int buf[5][2][512];
  __shared__ int rows_s[512];
  const int g = threadIdx.x;
  if (zero && g < nzero) zero[g] = 0;
  const int G = Eloc + S;
  int rows = 0;
  if (g < Eloc) rows = offsets[g + 1] - offsets[g];
  else if (g < G) rows = Tn;
  // bm1 tiles: a last m-tile with at most half its rows is a tail, counted apart
  const int rem1 = rows % bm1, is_tail = (rem1 > 0 && 2 * rem1 <= bm1) ? 1 : 0;
  buf[0][0][g] = (rows + bm0 - 1) / bm0;
  buf[1][0][g] = (rows + bm1 - 1) / bm1;
  buf[2][0][g] = (rows + bm1 - 1) / bm1 - is_tail;
  buf[3][0][g] = is_tail;
  buf[4][0][g] = (rows + bm2 - 1) / bm2;
  rows_s[g] = rows;
  __syncthreads();
  if (g < G) {
    int rank = 0;
    for (int h = 0; h < G; ++h) rank += (rows_s[h] > rows) || (rows_s[h] == rows && h < g);
    order[rank] = g;
  }
  if (g == 0) {  // order[G] = 1 when every group's row count is within 25% of the largest
    int lo = rows_s[0], hi = rows_s[0];
    for (int h = 1; h < G; ++h) {
      lo = min(lo, rows_s[h]);
      hi = max(hi, rows_s[h]);
    }
    order[G] = (G > 0 && 4 * hi <= 5 * lo) ? 1 : 0;
  }
  int cur = 0;
  for (int off = 1; off < 512; off <<= 1) {
#pragma unroll
    for (int w = 0; w < 5; ++w) {
      int x = buf[w][cur][g];
      if (g >= off) x += buf[w][cur][g - off];
      buf[w][cur ^ 1][g] = x;
    }
    cur ^= 1;
    __syncthreads();
  }
  if (g <= G) {
    pre0[g] = (g == 0) ? 0 : buf[0][cur][g - 1];
    pre1[g] = (g == 0) ? 0 : buf[1][cur][g - 1];
    body1[g] = (g == 0) ? 0 : buf[2][cur][g - 1];
    tail1[g] = (g == 0) ? 0 : buf[3][cur][g - 1];
    pre2[g] = (g == 0) ? 0 : buf[4][cur][g - 1];
  }
}

// ------------------------------------------------------------------------- host side

constexpr int T_BM = 128, T_BN = 128, T_WM = 2, T_WN = 2;

template <typename T, int KIND>
static hipError_t run_gemm(const GemmArgs& a, int grid, hipStream_t s, const char* name) {
  using Cf = TileCfg<T, T_BM, T_BN, T_WM, T_WN>;
  auto kern = grouped_gemm_kernel<T, T_BM, T_BN, T_WM, T_WN, KIND>;
  static std::atomic<uint64_t> lds_set{0};
  if (hipError_t e = lds_limit_once((const void*)kern, Cf::LDS, lds_set); e != hipSuccess) return e;
  if (grid <= 0) return hipSuccess;
  KernelTimer kt(name, s);
  hipLaunchKernelGGL(kern, dim3(grid), dim3(Cf::NT), Cf::LDS, s, a);
  return hipGetLastError();
}

static int round8(long v) { return (int)((v + 7) / 8 * 8); }

// Upper bound on the m-tiles of the row-ragged kinds (per-expert counts stay on the device).
static long mtile_bound(const moe_desc& d) {
  long routed = ((long)d.T * d.top_k + (long)d.local_count * (T_BM - 1)) / T_BM;
  return routed + (long)d.n_shared * ((d.T + T_BM - 1) / T_BM);
}

static GemmArgs base_args(const moe_desc& d, const int32_t* offsets, const int32_t* pre) {
  GemmArgs a{};
  a.T = d.T; a.k = d.top_k; a.d = d.d_model; a.f = d.d_ff; a.Eloc = d.local_count; a.S = d.n_shared;
  a.rows_cap = d.T * d.top_k;
  a.offsets = offsets;
  a.mt_prefix = pre;
  return a;
}

// pre: m-tile prefix for 128-row tiles (computed by the caller's plan launch)
hipError_t ffn_fwd_f32(const moe_desc& d, const void* x, const void* xp, const int32_t* offsets, const void* wg,
                       const void* wu, const void* wd, void* yp, void* saved, int32_t* pre, hipStream_t s) {
  using T = float;
  const size_t R = (size_t)rows_total(d), es = sizeof(T);
  GemmArgs a = base_args(d, offsets, pre);
  a.x = x; a.xp = xp; a.wg = wg; a.wu = wu; a.wd = wd;
  a.gu = saved;
  a.h = (char*)saved + align256(R * 2 * d.d_ff * es);
  a.out = yp;
  const long mtb = mtile_bound(d);
  hipError_t e;
  a.n_tiles = d.d_ff / (T_BN / 2);
  if ((e = run_gemm<T, FWD_GU>(a, round8(mtb * a.n_tiles), s, "gemm_fwd_gate_up")) != hipSuccess) return e;
  a.n_tiles = d.d_model / T_BN;
  if ((e = run_gemm<T, FWD_DOWN>(a, round8(mtb * a.n_tiles), s, "gemm_fwd_down")) != hipSuccess) return e;
  return hipGetLastError();
}

hipError_t ffn_bwd_f32(const moe_desc& d, const void* x, const void* xp, const void* dy, const void* dyp,
                       const int32_t* offsets, const void* wg, const void* wu, const void* wd, const void* saved,
                       void* dxp, void* dwg, void* dwu, void* dwd, void* dgu, int32_t* pre, hipStream_t s) {
  using T = float;
  const size_t R = (size_t)rows_total(d), es = sizeof(T);
  GemmArgs a = base_args(d, offsets, pre);
  a.x = x; a.xp = xp; a.dy = dy; a.dyp = dyp; a.wg = wg; a.wu = wu; a.wd = wd;
  a.gu = (void*)saved;
  a.h = (char*)saved + align256(R * 2 * d.d_ff * es);
  a.dgu = dgu;
  const long mtb = mtile_bound(d);
  const int G = d.local_count + d.n_shared;
  hipError_t e;
  a.n_tiles = d.d_ff / T_BN;
  if ((e = run_gemm<T, BWD_DH>(a, round8(mtb * a.n_tiles), s, "gemm_bwd_dh")) != hipSuccess) return e;
  a.out = dwd;
  a.m_tiles = d.d_model / T_BM;
  a.n_tiles = d.d_ff / T_BN;
  if ((e = run_gemm<T, WG_DOWN>(a, round8((long)G * a.m_tiles * a.n_tiles), s, "gemm_wgrad_down")) != hipSuccess)
    return e;
  a.out = dwg;
  a.out2 = dwu;
  a.m_tiles = 2 * d.d_ff / T_BM;
  a.n_tiles = d.d_model / T_BN;
  if ((e = run_gemm<T, WG_GU>(a, round8((long)G * a.m_tiles * a.n_tiles), s, "gemm_wgrad_gate_up")) != hipSuccess)
    return e;
  a.out = dxp;
  a.n_tiles = d.d_model / T_BN;
  if ((e = run_gemm<T, BWD_DX>(a, round8(mtb * a.n_tiles), s, "gemm_bwd_dx")) != hipSuccess) return e;
  return hipGetLastError();
}

}  // namespace pcmoe
