// Shared definitions of the HIP library (host and device).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "foremoe.h"

namespace foremoe {

// Pairs handled by one workgroup of the histogram and rank kernels. The two
// kernels must agree: the rank kernel starts each block from the prefix of
// the histogram's per-block counts.
constexpr int kHistChunk = 512;
constexpr int kHistThreads = 256;
constexpr int kWsHeaderBytes = 256;
// status word used internally as the arrival ticket of foremoe_histogram_assign
constexpr int kWsTicketWord = 63;

constexpr size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// Workspace layout (fixed offsets, so that every call can find its part
// from its own arguments). With a per-source plan the ranking keys are
// (source, expert) pairs, key = s * E + e, and slots are split the same way
// into virtual slots j * n_src + s; "keys" below is E or n_src * E.
//   [0, 256)                 int32 status words
//   [256, +64 KiB)           rep_slot[keys * R_max]: (virtual) slot of replica (key, r) or -1
//   [kWsVSlotOff, +4 KiB+4)  vslot_offset[S * n_src + 1]: row offsets of the virtual slots
//   [kWsPartialOff, ...)     per-block histogram partials [NB][keys+1]; the scan
//                            turns them into exclusive block bases
//   [ws_rank_off(), ...)     uint16 rank of every pair within its block's list
//                            of the same key [T*K] (written by the count kernel)
constexpr size_t kWsRepSlotOff = kWsHeaderBytes;
constexpr size_t kWsVSlotOff =
    kWsRepSlotOff + sizeof(int32_t) * (size_t)FOREMOE_MAX_EXPERTS * (size_t)FOREMOE_MAX_REPLICAS;
constexpr size_t kWsPartialOff = kWsVSlotOff + align_up(sizeof(int32_t) * ((size_t)FOREMOE_MAX_SLOTS + 1), 256);

inline int64_t hist_blocks(int64_t npairs) {
  int64_t nb = (npairs + kHistChunk - 1) / kHistChunk;
  return nb < 1 ? 1 : nb;
}

inline size_t ws_rank_off(int64_t T, int32_t K, int32_t E) {
  const int64_t nb = hist_blocks(T * (int64_t)K);
  return align_up(kWsPartialOff + sizeof(int32_t) * (size_t)nb * (size_t)(E + 1), 256);
}

inline size_t ws_bytes_needed(int64_t T, int32_t K, int32_t E) {
  return align_up(ws_rank_off(T, K, E) + sizeof(uint16_t) * (size_t)(T * (int64_t)K), 256);
}

// ---------------------------------------------------------------------------
// bfloat16 <-> float on the device (raw 16-bit patterns)
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf2f(uint32_t b16) { return __uint_as_float(b16 << 16); }

__device__ __forceinline__ uint32_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return 0x7FC0u;  // NaN
  u += 0x7FFFu + ((u >> 16) & 1u);  // round to nearest, ties to even
  return u >> 16;
}

__device__ __forceinline__ uint32_t pack_bf2(float lo, float hi) { return f2bf(lo) | (f2bf(hi) << 16); }

// Lanes below this one in a 64-bit lane mask.
__device__ __forceinline__ int lanes_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0));
}

__device__ __forceinline__ int lane_id() { return __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0)); }

// Deterministic butterfly sum over the 64 lanes of a wavefront.
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

}  // namespace foremoe

// ---------------------------------------------------------------------------
// Host-side error plumbing (defined in api.hip)
// ---------------------------------------------------------------------------
namespace foremoe {
int set_error(int status, const char* fmt, ...);
int check_launch(const char* what);
int num_cus();
}  // namespace foremoe
