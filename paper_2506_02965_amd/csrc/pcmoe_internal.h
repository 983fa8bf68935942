// Private helpers of the pcmoe HIP library (gfx950 / CDNA4). Not part of the ABI.
#pragma once
#include <atomic>
#include <type_traits>
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

#include "../../include/pcmoe.h"

namespace pcmoe {

typedef uint16_t bf16;  // bfloat16 storage (upper half of an IEEE binary32)
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

// 16-byte chunk: the unit of every global and LDS transfer of the hot kernels.
struct __align__(16) Chunk {
  uint32_t w[4];
};

__device__ __forceinline__ float bf2f(bf16 v) { return __uint_as_float(((uint32_t)v) << 16); }

// float -> bfloat16, round to nearest, ties to even (finite values).
// fp32 -> bf16, round to nearest even: one v_cvt_pk_bf16_f32 per pair of values on gfx950.
typedef __bf16 bf16x2_hw __attribute__((ext_vector_type(2)));
typedef float floatx2_hw __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((floatx2_hw){lo, hi}, bf16x2_hw));
}
__device__ __forceinline__ bf16 f2bf(float f) { return (bf16)(pack_bf16x2(f, 0.f) & 0xffffu); }

__device__ __forceinline__ float to_f(float v) { return v; }
__device__ __forceinline__ float to_f(bf16 v) { return bf2f(v); }
template <typename T> __device__ __forceinline__ T from_f(float v);
template <> __device__ __forceinline__ float from_f<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16 from_f<bf16>(float v) { return f2bf(v); }

// Elements of type T in one 16-byte chunk.
template <typename T> struct EPC;
template <> struct EPC<float> { static constexpr int value = 4; };
template <> struct EPC<bf16> { static constexpr int value = 8; };

// Unpack / pack a chunk to / from fp32 values.
template <typename T> __device__ __forceinline__ void chunk_to_f(const Chunk& c, float* out);
template <> __device__ __forceinline__ void chunk_to_f<float>(const Chunk& c, float* out) {
#pragma unroll
  for (int i = 0; i < 4; ++i) out[i] = __uint_as_float(c.w[i]);
}
template <> __device__ __forceinline__ void chunk_to_f<bf16>(const Chunk& c, float* out) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    out[2 * i] = __uint_as_float(c.w[i] << 16);
    out[2 * i + 1] = __uint_as_float(c.w[i] & 0xffff0000u);
  }
}
template <typename T> __device__ __forceinline__ Chunk f_to_chunk(const float* in);
template <> __device__ __forceinline__ Chunk f_to_chunk<float>(const float* in) {
  Chunk c;
#pragma unroll
  for (int i = 0; i < 4; ++i) c.w[i] = __float_as_uint(in[i]);
  return c;
}
template <> __device__ __forceinline__ Chunk f_to_chunk<bf16>(const float* in) {
  Chunk c;
#pragma unroll
  for (int i = 0; i < 4; ++i) c.w[i] = pack_bf16x2(in[2 * i], in[2 * i + 1]);
  return c;
}

__device__ __forceinline__ Chunk ld_chunk(const void* p) { return *reinterpret_cast<const Chunk*>(p); }
__device__ __forceinline__ void st_chunk(void* p, const Chunk& c) { *reinterpret_cast<Chunk*>(p) = c; }
// The same store marked non-temporal: for outputs that no kernel reads soon (weight gradients, the saved G|U), so
// that they do not push out of the last-level cache what the next kernels read.
__device__ __forceinline__ void st_chunk_nt(void* p, const Chunk& c) {
  typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
  const u32x4 v = {c.w[0], c.w[1], c.w[2], c.w[3]};
  __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(p));
}
__device__ __forceinline__ Chunk zero_chunk() {
  Chunk c;
  c.w[0] = c.w[1] = c.w[2] = c.w[3] = 0u;
  return c;
}

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
  return v;
}

// ---------------------------------------------------------------- host side

// Per-token row kernels are instantiated for KM = top_k rounded up to 1, 2, 4 or 8 and CPL = 16-byte chunks
// per lane per pass (1, 2 or 4: a row of cpr chunks takes ceil(cpr / (64 CPL)) passes). f(km, cpl) receives
// both as std::integral_constant.
template <typename F>
inline void row_dispatch(int k, int cpr, F&& f) {
  auto with_km = [&](auto km) {
    if (cpr <= 64) f(km, std::integral_constant<int, 1>{});
    else if (cpr <= 128) f(km, std::integral_constant<int, 2>{});
    else f(km, std::integral_constant<int, 4>{});
  };
  if (k <= 1) with_km(std::integral_constant<int, 1>{});
  else if (k <= 2) with_km(std::integral_constant<int, 2>{});
  else if (k <= 4) with_km(std::integral_constant<int, 4>{});
  else with_km(std::integral_constant<int, 8>{});
}

// Per-token row kernels that load several rows of a token at once: KM = top_k rounded up to 1, 2, 4, 6 or 8,
// SM = min(n_shared, 2) shared-expert rows loaded with them, and whether a router term is added (DL). f receives
// the three as std::integral_constant / std::bool_constant.
template <typename F>
inline void batch_dispatch(int k, int S, bool dl, F&& f) {
  auto with_sm = [&](auto km) {
    auto with_dl = [&](auto sm) {
      if (dl) f(km, sm, std::bool_constant<true>{});
      else f(km, sm, std::bool_constant<false>{});
    };
    if (S <= 0) with_dl(std::integral_constant<int, 0>{});
    else if (S == 1) with_dl(std::integral_constant<int, 1>{});
    else with_dl(std::integral_constant<int, 2>{});
  };
  if (k <= 1) with_sm(std::integral_constant<int, 1>{});
  else if (k <= 2) with_sm(std::integral_constant<int, 2>{});
  else if (k <= 4) with_sm(std::integral_constant<int, 4>{});
  else if (k <= 6) with_sm(std::integral_constant<int, 6>{});
  else with_sm(std::integral_constant<int, 8>{});
}
// 16-byte chunks per lane per pass for a kernel that keeps `rows` rows' chunks in flight at once (at most 32
// chunks, 128 VGPRs, of loads per lane).
constexpr int chunks_per_lane(int rows) { return rows <= 8 ? 4 : (rows <= 16 ? 2 : 1); }

// Bracket a kernel launch with HIP events when per-kernel timing is on (no-op otherwise).
struct KernelTimer {
  KernelTimer(const char* name, hipStream_t s);
  ~KernelTimer();
  const char* name;
  hipStream_t stream;
  void* slot;
};

// Raises a kernel's dynamic-LDS limit to `bytes` the first time it is launched on a device. `done` (one per
// kernel) holds a bit per device index below 64; concurrent first calls both set the same value, which is
// harmless. Returns hipSuccess or the runtime's error (then retried on the next call).
inline hipError_t lds_limit_once(const void* kern, int bytes, std::atomic<uint64_t>& done) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) dev = 0;
  const uint64_t bit = (dev >= 0 && dev < 64) ? (uint64_t)1 << dev : 0;
  if (bit && (done.load(std::memory_order_acquire) & bit)) return hipSuccess;
  const hipError_t e = hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  if (e == hipSuccess) done.fetch_or(bit, std::memory_order_release);
  return e;
}

// Launchers (defined next to their kernels). All return hipSuccess or the launch error.
hipError_t launch_route_fwd(const moe_desc& d, const void* x, const void* wr, const float* bias, int bias_groups,
                            float* logits, int32_t* idx, float* w, hipStream_t s);
hipError_t launch_route_bwd(const moe_desc& d, const void* x, const float* logits, const int32_t* idx,
                            const float* w, const float* dgate, float* dlogits, float* dwr, void* ws,
                            hipStream_t s);
size_t route_bwd_ws_bytes(const moe_desc& d);

hipError_t launch_permute(const moe_desc& d, const int32_t* idx, const void* x, int32_t* counts, int32_t* offsets,
                          int32_t* r2s, int32_t* s2r, void* xp, void* ws, hipStream_t s);
size_t permute_ws_bytes(const moe_desc& d);
size_t permute_noalloc_capacity();                // bytes of the fixed scratch of moe_permute_noalloc
hipError_t permute_noalloc_scratch(void** out);   // its device address on the current device
hipError_t launch_permute_bwd(const moe_desc& d, const void* dxp, const int32_t* s2r, const float* dlogits,
                              const void* wr, void* dx, hipStream_t s);

hipError_t launch_combine(const moe_desc& d, const void* yp, const int32_t* s2r, const float* w, void* y,
                          hipStream_t s);
hipError_t launch_combine_bwd(const moe_desc& d, const void* dy, const void* yp, const int32_t* s2r,
                              const float* w, void* dyp, float* dgate, hipStream_t s);

hipError_t launch_expert_update(const moe_desc& d, const moe_opt& o, void* wg, void* wu, void* wd, const void* gg,
                                const void* gu, const void* gd, float* master, float* m, float* v, hipStream_t s);

size_t ffn_saved_bytes(const moe_desc& d);
size_t ffn_fwd_ws_bytes(const moe_desc& d);
size_t ffn_bwd_ws_bytes(const moe_desc& d);
hipError_t launch_ffn_fwd(const moe_desc& d, const void* x, const void* xp, const int32_t* offsets,
                          const void* wg, const void* wu, const void* wd, void* yp, void* saved, void* ws,
                          hipStream_t s);
hipError_t launch_ffn_bwd(const moe_desc& d, const void* x, const void* xp, const void* dy, const void* dyp,
                          const int32_t* offsets, const void* wg, const void* wu, const void* wd,
                          const void* saved, void* dxp, void* dwg, void* dwu, void* dwd, void* ws,
                          hipStream_t s);

inline size_t elem_bytes(const moe_desc& d) { return d.dtype == MOE_BF16 ? 2 : 4; }
inline size_t align256(size_t v) { return (v + 255) & ~size_t(255); }
inline int64_t rows_total(const moe_desc& d) {
  return (int64_t)d.T * d.top_k + (int64_t)d.n_shared * d.T;
}

}  // namespace pcmoe
