// Step 4: grouped SwiGLU expert FFN over the local slots (App. A), forward,
// input gradient and weight gradient.
//
// bf16 path: persistent workgroups of 8 wavefronts (4 for 128-wide output
// tiles) walk a tile list built on the device from the slot offsets (no
// host sync). Operand tiles stream from
// HBM straight into LDS with range-checked buffer loads (buffer_load ... lds:
// no staging registers; rows outside the current slot read as zero and no
// load can leave its operand) through a ring of LDS stages, and are
// multiplied with v_mfma_f32_32x32x16_bf16 (fp32 accumulation). Operands
// that are contiguous along K are read with ds_read_b128; operands contiguous
// along M/N (the weights in dgrad, both operands of wgrad) stay in their
// memory layout in LDS and are read with the gfx950 transpose read
// ds_read_b64_tr_b16. The SwiGLU activation and its derivative are fused into
// the epilogues.
//
// f32 path: plain per-element kernels (small shapes only; no MFMA).
#include <climits>
#include <type_traits>

#include "common.h"

namespace foremoe {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

// Tile configurations (overridable at build time for tuning sweeps).
#ifndef FM_ROWS_BK
#define FM_ROWS_BK 64
#endif
#ifndef FM_ROWS_NS
#define FM_ROWS_NS 2
#endif
#ifndef FM_ROWS_WGM
#define FM_ROWS_WGM 4
#endif
#ifndef FM_ROWS_WGN
#define FM_ROWS_WGN 2
#endif
#ifndef FM_WG_BK
#define FM_WG_BK 64
#endif
#ifndef FM_WG_NS
#define FM_WG_NS 2
#endif
#ifndef FM_WG_WGM
#define FM_WG_WGM 2
#endif
#ifndef FM_WG_WGN
#define FM_WG_WGN 4
#endif
// k-steps over which one stage's loads are spread (capped at the k-steps of a stage)
#ifndef FM_LOAD_SPREAD
#define FM_LOAD_SPREAD 2
#endif
// Wave priority while a k-step's MFMAs issue (0: leave it): the wave that
// is multiplying wins the SIMD's issue arbitration over the other wave on
// that SIMD, whose reads and loads then fill the gaps.
#ifndef FM_SETPRIO
#define FM_SETPRIO 1
#endif

enum Epi { kEpiStore = 0, kEpiSwigluFwd = 1, kEpiSwigluBwd = 2 };

__device__ __forceinline__ float silu_f(float a) { return a / (1.0f + __expf(-a)); }

__device__ __forceinline__ int lane64() { return threadIdx.x & 63; }
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

// Virtual workgroup id: workgroups are dispatched round-robin over the 8 XCDs,
// so give the workgroups of one XCD consecutive ids (they then share tiles
// that reuse the same operand rows in that XCD's L2).
#ifndef FM_XCD_MAP
#define FM_XCD_MAP 1
#endif
__device__ __forceinline__ int xcd_virtual_id() {
  const int b = blockIdx.x, n = gridDim.x;
  if (!FM_XCD_MAP || n % 8 != 0) return b;
  return (b % 8) * (n / 8) + b / 8;
}

// Block-wide inclusive scan (up to 16 wavefronts; s_tmp holds one int per wave).
__device__ int block_scan(int v, int* s_tmp, int& total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int n = __shfl_up(v, o, 64);
    if (lane >= o) v += n;
  }
  if (lane == 63) s_tmp[w] = v;
  __syncthreads();
  int before = 0;
  total = 0;
  for (int i = 0; i < nw; ++i) {
    const int t = s_tmp[i];
    if (i < w) before += t;
    total += t;
  }
  __syncthreads();
  return v + before;
}

// ---------------------------------------------------------------------------
// Range-checked buffer loads straight into LDS
// ---------------------------------------------------------------------------
// A buffer resource over [base, base + bytes): a load at an offset >= bytes
// returns zeros, so ragged tile edges read as zero and no load can leave the
// operand.
__device__ __forceinline__ i32x4 buf_rsrc(const void* base, uint32_t bytes) {
  const uint64_t a = (uint64_t)base;
  i32x4 r;
  r.x = __builtin_amdgcn_readfirstlane((int)(uint32_t)a);
  r.y = __builtin_amdgcn_readfirstlane((int)((a >> 32) & 0xFFFFu));
  r.z = __builtin_amdgcn_readfirstlane((int)bytes);
  r.w = 0x00020000;
  return r;
}

// One wavefront moves 64 x 16 bytes: lane l's bytes land at LDS address
// lds_wave_base + 16 l. The load is issued asynchronously; completion is
// awaited with wait_vm() before the workgroup barrier that publishes it.
__device__ __forceinline__ void dma16(i32x4 rs, uint32_t lds_wave_base, uint32_t voff) {
  const uint32_t m0v = __builtin_amdgcn_readfirstlane(lds_wave_base);
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds" ::"s"(m0v), "v"(voff), "s"(rs)
               : "memory");
}

// The same with lane offset voff0 + soff (soff wave-uniform): the add sits
// in the asm so that one temporary serves every load instead of one
// precomputed offset register per load.
__device__ __forceinline__ void dma16s(i32x4 rs, uint32_t lds_wave_base, uint32_t voff0, uint32_t soff) {
  const uint32_t m0v = __builtin_amdgcn_readfirstlane(lds_wave_base);
  uint32_t t;
  asm volatile(
      "v_add_u32 %0, %1, %2\n\ts_mov_b32 m0, %3\n\tbuffer_load_dwordx4 %0, %4, 0 offen lds"
      : "=&v"(t)
      : "s"(soff), "v"(voff0), "s"(m0v), "s"(rs)
      : "memory");
}

// Wait until at most N vector-memory operations of this wavefront are in flight.
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

__device__ __forceinline__ uint32_t lds_addr(const void* p) { return (uint32_t)(uintptr_t)p; }

// ---------------------------------------------------------------------------
// LDS operand tiles. A "K-major" tile keeps ROWS rows (m or n) of BK
// contiguous k values; a "MN-major" tile keeps BK rows (k) of ROWS contiguous
// m or n values. Both are filled by dma16 and XOR-swizzled in 16-byte chunks
// so that the MFMA fragment reads hit 16 (or 32) different LDS bank groups of
// gfx950's 64 banks.
// ---------------------------------------------------------------------------
template <int ROWS, int BK, int NW>
struct KTile {
  static constexpr int CPR = BK / 8;     // 16-byte chunks per row
  static constexpr int RPI = 64 / CPR;   // rows per wavefront load
  static constexpr int NI = ROWS / RPI;  // wavefront loads per tile
  static constexpr int PER_WAVE = NI / NW;
  static constexpr int BYTES = ROWS * BK * 2;
  static_assert(NI % NW == 0, "tile must split over the wavefronts");
  __device__ __forceinline__ static int swz(int r) {
    if constexpr (CPR == 8) return (r >> 1) & 7;
    else return (r >> 2) & 3;
  }
  // This lane's source offset in load i (0 <= i < PER_WAVE) of this
  // wavefront's share of the tile, relative to the stage's first k; rowoff(r)
  // is the byte offset of tile row r. Fixed for a whole tile: each stage
  // moves the buffer resource instead.
  template <class RowOff>
  __device__ __forceinline__ static uint32_t voff(RowOff rowoff, int i) {
    const int l = lane64(), w = wave_id();
    const int r = (w + NW * i) * RPI + l / CPR;
    const int c = (l % CPR) ^ swz(r);
    return rowoff(r) + (uint32_t)c * 16u;
  }
  __device__ __forceinline__ static void issue(i32x4 rs, uint32_t lds, uint32_t voff, int i) {
    dma16(rs, lds + (wave_id() + NW * i) * 1024, voff);
  }
  // load i with lane offset voff(0) + soff_i, soff_i = voff(i) - voff(0) (the
  // same for every lane: the swizzle of a row or k row does not change by i)
  __device__ __forceinline__ static void issue_s(i32x4 rs, uint32_t lds, uint32_t voff0, uint32_t soff, int i) {
    dma16s(rs, lds + (wave_id() + NW * i) * 1024, voff0, soff);
  }
  // MFMA operand for rows mn0..mn0+31 of the tile, k-step kk (16 k values):
  // lane l gets row mn0 + l % 32, k = 16 kk + 8 (l / 32) + 0..7. The swizzle
  // only depends on l % 32 (mn0 is a multiple of 32), so the address splits
  // into a per-block lane offset and a per-k-step lane offset.
  __device__ __forceinline__ static uint32_t lane_off(int mn0) {
    return (uint32_t)(mn0 + (lane64() & 31)) * (BK * 2);
  }
  __device__ __forceinline__ static uint32_t kstep_off(int kk) {
    const int l = lane64();
    return (uint32_t)(((2 * kk + (l >> 5)) ^ swz(l & 31)) * 16);
  }
  __device__ __forceinline__ static bf16x8 frag(const char* lds, uint32_t off, const uint32_t* koff, int kk) {
    return *reinterpret_cast<const bf16x8*>(lds + off + koff[kk]);
  }
};

template <int ROWS, int BK, int NW>
struct MTile {
  static constexpr int RB = ROWS * 2;    // bytes per k row
  static constexpr int KPI = 1024 / RB;  // k rows per wavefront load
  static constexpr int NI = BK / KPI;
  static constexpr int PER_WAVE = NI / NW;
  static constexpr int BYTES = ROWS * BK * 2;
  static_assert(NI % NW == 0 && KPI >= 1, "tile must split over the wavefronts");
  __device__ __forceinline__ static int swz(int k) { return 4 * (k & 3); }
  // This lane's source offset in load i (0 <= i < PER_WAVE) of this
  // wavefront's share of the tile; koff(k) is the byte offset of the tile's
  // k-row k (relative to the stage's first k row) at the tile's first m/n.
  template <class KOff>
  __device__ __forceinline__ static uint32_t voff(KOff koff, int i) {
    const int l = lane64(), w = wave_id();
    const int k = (w + NW * i) * KPI + (l * 16) / RB;
    const int c = ((l * 16) % RB) / 16 ^ swz(k);
    return koff(k) + (uint32_t)c * 16u;
  }
  __device__ __forceinline__ static void issue(i32x4 rs, uint32_t lds, uint32_t voff, int i) {
    dma16(rs, lds + (wave_id() + NW * i) * 1024, voff);
  }
  // load i with lane offset voff(0) + soff_i, soff_i = voff(i) - voff(0) (the
  // same for every lane: the swizzle of a row or k row does not change by i)
  __device__ __forceinline__ static void issue_s(i32x4 rs, uint32_t lds, uint32_t voff0, uint32_t soff, int i) {
    dma16s(rs, lds + (wave_id() + NW * i) * 1024, voff0, soff);
  }
  // Same operand layout as KTile::frag, assembled from two transpose reads:
  // in each 16-lane group g, lane i addresses 4 consecutive m/n of one k row
  // and lane j receives one m/n at 4 consecutive k. The k row's low two bits
  // (which pick the swizzle) come from the lane alone, so the address is a
  // per-block lane offset plus an immediate (16 kk + 4 h) * RB.
  __device__ __forceinline__ static uint32_t lane_off(int mn0) {
    const int l = lane64();
    const int g = l >> 4, j = l & 15;
    const int krow = 8 * (g >> 1) + (j >> 2);
    const int mn = mn0 + 16 * (g & 1) + 4 * (j & 3);
    return (uint32_t)(krow * RB + (((mn >> 3) ^ swz(krow)) << 4) + (mn & 7) * 2);
  }
  __device__ __forceinline__ static uint32_t kstep_off(int) { return 0; }
  __device__ __forceinline__ static bf16x8 frag(const char* lds, uint32_t off, const uint32_t*, int kk) {
    s16x4 v[2];
#pragma unroll
    for (int h = 0; h < 2; ++h)
      v[h] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(lds + off + (kk * 16 + 4 * h) * RB));
    const s16x8 t = __builtin_shufflevector(v[0], v[1], 0, 1, 2, 3, 4, 5, 6, 7);
    return __builtin_bit_cast(bf16x8, t);
  }
};

// ---------------------------------------------------------------------------
// MFMA tile core: WGM x WGN wavefronts, each owning (BM/WGM) x (BN/WGN) of
// the output as 32x32 blocks. The MFMA is fed the B rows as its first
// operand, so each lane ends up with 4 consecutive output columns of one
// output row: block (i, j), register q of lane l holds row
// wm*WM + 32 i + l % 32 and column bcol(j) + 8 (q / 4) + 4 (l / 32) + q % 4.
// ---------------------------------------------------------------------------
template <int BM, int BN, int WGM, int WGN, bool SWIGLU_COLS>
struct Core {
  static constexpr int WM = BM / WGM, WN = BN / WGN;
  static constexpr int MB = WM / 32, NB = WN / 32;
  static constexpr int GW = BN / 2 / WGN;  // SwiGLU: gate (or up) columns per wave
  static_assert(MB >= 1 && NB >= 1 && (!SWIGLU_COLS || NB % 2 == 0), "wave tile");
  f32x16 acc[MB][NB];

  // LDS row of the B tile that wave column wn's block j starts at.
  __device__ __forceinline__ static int bcol(int wn, int j) {
    if constexpr (SWIGLU_COLS) {
      // gate rows live in [0, BN/2), up rows in [BN/2, BN); the wave keeps the
      // gate block j and the up block j + NB/2 of the same output columns
      constexpr int H = NB / 2;
      return j < H ? wn * GW + j * 32 : BN / 2 + wn * GW + (j - H) * 32;
    } else {
      return wn * WN + j * 32;
    }
  }

  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
      for (int j = 0; j < NB; ++j)
#pragma unroll
        for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.f;
  }

  // Per-lane LDS offsets of every 32-row block this wave reads (fixed for
  // the whole kernel) and of every k-step.
  template <class AT, class BT, int BK>
  struct Offsets {
    uint32_t a[MB], b[NB], ka[BK / 16], kb[BK / 16];
    __device__ __forceinline__ Offsets(int wm, int wn) {
#pragma unroll
      for (int i = 0; i < MB; ++i) a[i] = AT::lane_off(wm * WM + i * 32);
#pragma unroll
      for (int j = 0; j < NB; ++j) b[j] = BT::lane_off(bcol(wn, j));
#pragma unroll
      for (int kk = 0; kk < BK / 16; ++kk) {
        ka[kk] = AT::kstep_off(kk);
        kb[kk] = BT::kstep_off(kk);
      }
    }
  };

  // Operand fragments of FS k-steps in registers (the one being multiplied
  // and the ones being read ahead).
  template <int FS>
  struct Frags {
    bf16x8 a[FS][MB], b[FS][NB];
  };

  template <class AT, class BT, int BK, class FragsT>
  __device__ __forceinline__ static void load_frags(FragsT& f, int set, const char* As, const char* Bs,
                                                    const Offsets<AT, BT, BK>& o, int kk) {
#pragma unroll
    for (int i = 0; i < MB; ++i) f.a[set][i] = AT::frag(As, o.a[i], o.ka, kk);
#pragma unroll
    for (int j = 0; j < NB; ++j) f.b[set][j] = BT::frag(Bs, o.b[j], o.kb, kk);
  }

  // The MFMAs of one k-step from register set CUR, with the LDS reads of a
  // later k-step's fragments (k-step nkk of the stage at nAs/nBs, into set
  // NXT) interleaved: one read after each of the first MB + NB MFMAs, so the
  // reads complete under the matrix work. extra(q), q < NX, runs right after
  // MFMA s when q < (s + 1) NX / (MB NB) and q >= s NX / (MB NB), evenly
  // over the k-step: the loads of a later stage, spread over the k-step so
  // that the address unit drains them while the matrix cores keep working.
  template <class AT, class BT, int BK, int NX, int CUR, int NXT, class FragsT, class Extra>
  __device__ __forceinline__ void mfma_step(FragsT& f, const char* nAs, const char* nBs, const Offsets<AT, BT, BK>& o,
                                            int nkk, Extra&& extra) {
    constexpr int NM = MB * NB;
    static_assert(NX >= 0 && NX <= NM, "loads per k-step");
    static_assert(CUR != NXT, "the fragments being read go to another set");
    if constexpr (FM_SETPRIO > 0) __builtin_amdgcn_s_setprio(FM_SETPRIO);
#pragma unroll
    for (int s = 0; s < NM; ++s) {
      const int i = s / NB, j = s % NB;
      acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.b[CUR][j], f.a[CUR][i], acc[i][j], 0, 0, 0);
      if (FM_SETPRIO > 0 && s == NM - 1) __builtin_amdgcn_s_setprio(0);
      if (s < MB + NB) {
        if (s < MB) f.a[NXT][s] = AT::frag(nAs, o.a[s], o.ka, nkk);
        else f.b[NXT][s - MB] = BT::frag(nBs, o.b[s - MB], o.kb, nkk);
      }
      if constexpr (NX > 0) {
#pragma unroll
        for (int q = s * NX / NM; q < (s + 1) * NX / NM; ++q) extra(q);
      }
    }
#pragma unroll
    for (int s = 0; s < NM; ++s) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
      if (s < MB + NB) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one LDS read
    }
  }

  template <class AT, class BT, int BK>
  __device__ __forceinline__ void compute(const char* As, const char* Bs, const Offsets<AT, BT, BK>& o) {
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      bf16x8 af[MB], bfr[NB];
#pragma unroll
      for (int i = 0; i < MB; ++i) af[i] = AT::frag(As, o.a[i], o.ka, kk);
#pragma unroll
      for (int j = 0; j < NB; ++j) bfr[j] = BT::frag(Bs, o.b[j], o.kb, kk);
#pragma unroll
      for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int j = 0; j < NB; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[j], af[i], acc[i][j], 0, 0, 0);
    }
  }
};

// Wait for the loads of the stage about to be computed: `ahead` younger
// stages (of PER loads each) may stay in flight.
template <int NS, int PER>
__device__ __forceinline__ void wait_stage(int ahead) {
  static_assert(NS >= 2 && NS <= 4 && (NS - 1) * PER < 64, "stages");
  if constexpr (NS >= 4) {
    if (ahead >= 3) {
      wait_vm<3 * PER>();
      return;
    }
  }
  if constexpr (NS >= 3) {
    if (ahead >= 2) {
      wait_vm<2 * PER>();
      return;
    }
  }
  if (ahead >= 1) {
    wait_vm<PER>();
    return;
  }
  wait_vm<0>();
}

// ---------------------------------------------------------------------------
// Software-pipelined K loop over an LDS ring of NS >= 2 stages.
//
// Stage kt's first fragments are already in registers when iteration kt
// starts, and every later k-step's fragments are read one k-step ahead. So
// when the last k-step of stage kt begins, every read of stage kt's buffer
// has been issued: each wavefront waits for its own loads of stage kt+1, and
// the workgroup barrier (which also retires all LDS reads) both publishes
// stage kt+1 and frees stage kt's buffer. The loads of stage kt+NS go into
// that buffer, spread over the MFMAs of the last k-step of stage kt and the
// first k-steps of stage kt+1 (issued in one burst, they would stall every
// wavefront behind the address unit at once). issue(s, p) issues load p
// (0 <= p < PER) of stage s, in increasing s, each stage whole before the
// next. Stages s >= KT must issue loads of nothing (zero-size buffer
// resources, which still write zeros to their LDS stage): every iteration
// then issues the same loads, with no branch among the MFMAs, and the
// counter waits stay exact.
// ---------------------------------------------------------------------------
template <int I, int N, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<I + 1, N>(f);
  }
}

// Fragment read distance of the row GEMMs: 2 for the gate/up forward (2%
// faster than 1 on the benchmark), 1 for the others (with a third register
// set they spill, and run 4-6% slower).
#ifndef FM_FRAG_DIST_FWD
#define FM_FRAG_DIST_FWD 2
#endif
#ifndef FM_FRAG_DIST
#define FM_FRAG_DIST 1
#endif

// Fragments read one k-step ahead (two register sets).
template <class CoreT, class AT, class BT, int BK, int NS, class Issue>
__device__ __forceinline__ void pipelined_k_loop_d1(CoreT& core, char* lds, int KT,
                                                    const typename CoreT::template Offsets<AT, BT, BK>& o,
                                                    Issue&& issue) {
  static_assert(BK % 32 == 0, "the last k-step's fragments must be read before the barrier");
  constexpr int KK = BK / 16;
  constexpr int STAGE = AT::BYTES + BT::BYTES;
  constexpr int PER = AT::PER_WAVE + BT::PER_WAVE;
  // the loads of a stage ride on SPREAD k-steps: the last one of the stage
  // before and the first SPREAD - 1 of the next; load p goes with k-step
  // j when lo(j) <= p < lo(j + 1)
  constexpr int SPREAD = FM_LOAD_SPREAD < KK ? FM_LOAD_SPREAD : KK;
  static_assert(SPREAD >= 1, "load spread");
  auto lo = [](int j) constexpr { return j * PER / SPREAD; };
  typename CoreT::template Frags<2> f;
  // stages 0 .. NS-2 whole, and the part of stage NS-1 that a previous
  // iteration's last k-step would have carried
#pragma unroll
  for (int s = 0; s < NS; ++s) {
#pragma unroll
    for (int p = 0; p < (s < NS - 1 ? PER : lo(1)); ++p) issue(s, p);
  }
  wait_vm<(NS - 2) * PER + lo(1)>();
  __syncthreads();
  CoreT::template load_frags<AT, BT, BK>(f, 0, lds, lds + AT::BYTES, o, 0);
  for (int kt = 0; kt < KT; ++kt) {
    const char* st = lds + (kt % NS) * STAGE;
    static_for<0, KK>([&](auto kkc) {
      constexpr int kk = decltype(kkc)::value;
      constexpr int set = kk & 1;
      if constexpr (kk < KK - 1) {
        constexpr int j = kk + 1;  // position in the load window of stage kt - 1 + NS
        core.template mfma_step<AT, BT, BK, (j < SPREAD ? lo(j + 1) - lo(j) : 0), set, set ^ 1>(
            f, st, st + AT::BYTES, o, kk + 1, [&](int q) { issue(kt - 1 + NS, lo(j) + q); });
      } else {
        wait_stage<NS, PER>(NS - 2);  // stage kt+1 (past the last: empty) has landed
        __syncthreads();
        const char* nst = lds + ((kt + 1) % NS) * STAGE;
        // (after the last stage this reads a stale buffer: harmless, and no
        // branch among the MFMAs)
        core.template mfma_step<AT, BT, BK, lo(1), set, set ^ 1>(f, nst, nst + AT::BYTES, o, 0,
                                                                 [&](int q) { issue(kt + NS, q); });
      }
    });
  }
  wait_vm<0>();  // the (empty) loads of stages past the last have landed too
}

// Fragments read D k-steps ahead (D + 1 register sets), so that each LDS read
// has D k-steps of matrix work to complete under. The barrier then comes at
// k-step KK - D of stage kt, the first whose reads reach into stage kt+1: by
// then every read of stage kt's buffer has been issued, and the loads of
// stage kt+NS go into it during k-steps KK - D .. KK - D + SPREAD - 1. The
// set of global k-step g is g % (D + 1); the stage loop is unrolled U times
// so that every set index is a compile-time constant.
template <class CoreT, class AT, class BT, int BK, int NS, int D, class Issue>
__device__ __forceinline__ void pipelined_k_loop_deep(CoreT& core, char* lds, int KT,
                                                      const typename CoreT::template Offsets<AT, BT, BK>& o,
                                                      Issue&& issue) {
  constexpr int KK = BK / 16;
  constexpr int FS = D + 1;
  constexpr int STAGE = AT::BYTES + BT::BYTES;
  constexpr int PER = AT::PER_WAVE + BT::PER_WAVE;
  constexpr int SPREAD = FM_LOAD_SPREAD < D ? FM_LOAD_SPREAD : D;
  static_assert(D >= 2 && KK >= D, "read distance");
  static_assert(SPREAD >= 1, "load spread");
  auto lo = [](int j) constexpr { return j * PER / SPREAD; };
  constexpr int U = [] {
    int u = 1;
    while ((u * KK) % FS) ++u;
    return u;
  }();
  typename CoreT::template Frags<FS> f;
#pragma unroll
  for (int s = 0; s < NS; ++s) {
#pragma unroll
    for (int p = 0; p < PER; ++p) issue(s, p);
  }
  wait_stage<NS, PER>(NS - 1);  // stage 0 has landed
  __syncthreads();
  static_for<0, D>([&](auto kc) {
    constexpr int k = decltype(kc)::value;
    CoreT::template load_frags<AT, BT, BK>(f, k, lds, lds + AT::BYTES, o, k);
  });
  int kt = 0;
  while (kt < KT) {  // kt advances inside the unrolled stage loop
    static_for<0, U>([&](auto phc) {
      constexpr int ph = decltype(phc)::value;
      if (kt >= KT) return;
      const char* st = lds + (kt % NS) * STAGE;
      const char* nst = lds + ((kt + 1) % NS) * STAGE;
      static_for<0, KK>([&](auto kkc) {
        constexpr int kk = decltype(kkc)::value;
        constexpr int g = ph * KK + kk;
        constexpr int cur = g % FS, nxt = (g + D) % FS;
        constexpr int j = kk - (KK - D);  // position in the load window of stage kt + NS
        constexpr int nx = (j >= 0 && j < SPREAD) ? lo(j + 1) - lo(j) : 0;
        if constexpr (j == 0) {
          wait_stage<NS, PER>(NS - 2);  // stage kt+1 (past the last: empty) has landed
          __syncthreads();
        }
        // reads of k-step kk + D: in this stage's buffer, or in the next's
        // (after the last stage a stale buffer: harmless, and no branch among
        // the MFMAs)
        const char* rs = kk + D < KK ? st : nst;
        constexpr int rk = (kk + D) % KK;
        core.template mfma_step<AT, BT, BK, nx, cur, nxt>(f, rs, rs + AT::BYTES, o, rk, [&](int q) {
          if constexpr (j >= 0) issue(kt + NS, lo(j) + q);
        });
      });
      ++kt;
    });
  }
  wait_vm<0>();  // the (empty) loads of stages past the last have landed too
}

template <class CoreT, class AT, class BT, int BK, int NS, int D = FM_FRAG_DIST, class Issue>
__device__ __forceinline__ void pipelined_k_loop(CoreT& core, char* lds, int KT,
                                                 const typename CoreT::template Offsets<AT, BT, BK>& o,
                                                 Issue&& issue) {
  if constexpr (D >= 2 && BK / 16 >= D)
    pipelined_k_loop_deep<CoreT, AT, BT, BK, NS, D>(core, lds, KT, o, issue);
  else
    pipelined_k_loop_d1<CoreT, AT, BT, BK, NS>(core, lds, KT, o, issue);
}

// ---------------------------------------------------------------------------
// Row-grouped GEMM: for each slot j, rows [off_j, off_{j+1}) (clamped to
// n_cap) times the slot's weight matrix.
// ---------------------------------------------------------------------------
struct RowsArgs {
  const uint16_t* A;  // [n_cap, K]
  int64_t lda;
  const uint16_t* B;  // weights; matrix w starts at B + w * wstride
  int64_t ldb;
  int64_t wstride;
  int W;
  int K;
  int N;   // output columns of the tile grid (2F for the fused gate/up)
  int F;   // SwiGLU width
  const int32_t* slot_offset;
  const int32_t* slot_widx;
  int S;
  int64_t n_cap;
  uint16_t* C;  // main output
  int64_t ldc;
  uint16_t* C2;  // forward: saved [A | U] or NULL
  int64_t ldc2;
  const uint16_t* AU;  // input gradient: saved [A | U]
  int64_t ldau;
  float* sk_part;      // split workspace: one partial tile per workgroup, or NULL
  unsigned* sk_count;  // arrival count per tile of the split round (zero between calls)
};

// Per-slot m-tile prefix in LDS: s_mt[j] = m-tiles of slots before j.
template <int BM>
__device__ void build_slot_tiles(const int32_t* __restrict__ off, int S, int64_t n_cap, int* s_mt, int* s_tmp) {
  int carry = 0;
  for (int j0 = 0; j0 < S; j0 += (int)blockDim.x) {
    const int j = j0 + threadIdx.x;
    int n = 0;
    if (j < S) {
      int64_t lo = off[j], hi = off[j + 1];
      lo = lo < 0 ? 0 : (lo > n_cap ? n_cap : lo);
      hi = hi < 0 ? 0 : (hi > n_cap ? n_cap : hi);
      n = hi > lo ? (int)((hi - lo + BM - 1) / BM) : 0;
    }
    int total;
    const int incl = block_scan(n, s_tmp, total);
    if (j < S) s_mt[j] = carry + incl - n;
    carry += total;
  }
  if (threadIdx.x == 0) s_mt[S] = carry;
  __syncthreads();
}

// ---------------------------------------------------------------------------
// Row-GEMM epilogue through LDS. The MFMA leaves each lane with 4-column
// pieces of 32 different rows; stored directly, every store instruction
// would touch 32 partly written lines. Instead each wavefront converts one
// 32-row block at a time to bf16 in its own LDS region and reads it back as
// whole row segments, 16 bytes per lane with consecutive lanes along a row,
// so each store instruction writes complete 128-byte lines. The staged rows
// are XOR-swizzled in 16-byte chunks so that the 8-byte writes of 32 rows
// spread over the LDS banks.
// ---------------------------------------------------------------------------
template <int RB>  // bytes per staged row
struct StagedRows {
  static constexpr int CPR = RB / 16;                   // 16-byte chunks per row
  static constexpr int RPB = RB >= 256 ? 1 : 256 / RB;  // rows per 256-byte bank cycle
  static constexpr int RPI = 64 / CPR;                  // rows per wavefront instruction
  static constexpr int NI = 32 / RPI;                   // instructions per 32-row block
  static constexpr int BYTES = 32 * RB;
  static_assert(CPR >= 1 && CPR <= 64 && 32 % RPI == 0, "staged row width");
  __device__ __forceinline__ static uint32_t chunk(int r, int c) {
    return (uint32_t)(r * RB + ((c ^ ((r / RPB) % CPR)) << 4));
  }
  // 4 consecutive values at column col (a multiple of 4) of row r
  __device__ __forceinline__ static void put4(char* base, int r, int col, float v0, float v1, float v2, float v3) {
    *reinterpret_cast<uint2*>(base + chunk(r, col >> 3) + ((col & 4) << 1)) =
        make_uint2(pack_bf2(v0, v1), pack_bf2(v2, v3));
  }
  // the 16-byte chunk lane l reads back in instruction it: row, chunk index
  __device__ __forceinline__ static int row_of(int it) { return it * RPI + lane64() / CPR; }
  __device__ __forceinline__ static int col_of() { return lane64() % CPR; }
  __device__ __forceinline__ static uint4 get(const char* base, int r, int c) {
    return *reinterpret_cast<const uint4*>(base + chunk(r, c));
  }
};

// fp32 staging (the SwiGLU backward keeps dH in fp32): RB bytes per row,
// 16-byte chunks of 4 floats; lane l reads back 8 consecutive floats.
template <int RB>
struct StagedRowsF32 {
  static constexpr int CPR = RB / 16;
  static constexpr int LPR = CPR / 2;  // lanes per row in the read-back
  static constexpr int RPI = 64 / LPR;
  static constexpr int NI = 32 / RPI;
  static constexpr int BYTES = 32 * RB;
  static_assert(RB % 256 == 0 && LPR >= 1 && LPR <= 64 && 32 % RPI == 0, "staged row width");
  __device__ __forceinline__ static uint32_t chunk(int r, int c) { return (uint32_t)(r * RB + ((c ^ (r % 16)) << 4)); }
  __device__ __forceinline__ static void put4(char* base, int r, int col, float v0, float v1, float v2, float v3) {
    *reinterpret_cast<float4*>(base + chunk(r, col >> 2)) = make_float4(v0, v1, v2, v3);
  }
  __device__ __forceinline__ static int row_of(int it) { return it * RPI + lane64() / LPR; }
  __device__ __forceinline__ static int col_of() { return lane64() % LPR; }  // in units of 8 values
  __device__ __forceinline__ static void get8(const char* base, int r, int c8, float* f) {
    const float4 lo = *reinterpret_cast<const float4*>(base + chunk(r, 2 * c8));
    const float4 hi = *reinterpret_cast<const float4*>(base + chunk(r, 2 * c8 + 1));
    f[0] = lo.x; f[1] = lo.y; f[2] = lo.z; f[3] = lo.w;
    f[4] = hi.x; f[5] = hi.y; f[6] = hi.z; f[7] = hi.w;
  }
};

template <class CoreT, int EPI>
struct EpiBytes {
  // SwiGLU forward stages H, A and U (GW bf16 columns each), the backward
  // WN fp32 columns, the plain store WN bf16 columns
  static constexpr int PER_WAVE = EPI == kEpiSwigluFwd   ? 3 * StagedRows<CoreT::GW * 2>::BYTES
                                  : EPI == kEpiSwigluBwd ? StagedRowsF32<CoreT::WN * 4>::BYTES
                                                         : StagedRows<CoreT::WN * 2>::BYTES;
};

__device__ __forceinline__ void unpack8(uint4 v, float* f) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = bf2f(w[i] & 0xFFFFu);
    f[2 * i + 1] = bf2f(w[i] >> 16);
  }
}

__device__ __forceinline__ uint4 pack8(const float* f) {
  return make_uint4(pack_bf2(f[0], f[1]), pack_bf2(f[2], f[3]), pack_bf2(f[4], f[5]), pack_bf2(f[6], f[7]));
}

// Writes this wave's output block: rows wrow0 .. wrow0 + WM - 1 (those below
// rend), output columns n0 + wn * WN .. (SwiGLU forward: H columns
// f0 + wn * GW ..). `ep` is the wave's private LDS region.
template <class CoreT, int EPI>
__device__ __forceinline__ void rows_epilogue(const RowsArgs& a, const CoreT& core, char* ep, int64_t wrow0,
                                              int64_t rend, int n0, int f0, int wn) {
  const int lane = lane64();
  const int l32 = lane & 31, c4 = (lane >> 5) * 4;
#pragma unroll
  for (int i = 0; i < CoreT::MB; ++i) {
    const int64_t prow0 = wrow0 + i * 32;
    if (prow0 >= rend) break;
    if constexpr (EPI == kEpiSwigluFwd) {
      using SR = StagedRows<CoreT::GW * 2>;
      constexpr int H = CoreT::NB / 2;
      char* sh = ep;
      char* sa = ep + SR::BYTES;
      char* su = ep + 2 * SR::BYTES;
#pragma unroll
      for (int jj = 0; jj < H; ++jj)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int col = jj * 32 + g * 8 + c4;
          float hv[4], av[4], uv[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            av[e] = core.acc[i][jj][g * 4 + e];
            uv[e] = core.acc[i][jj + H][g * 4 + e];
            hv[e] = silu_f(av[e]) * uv[e];
          }
          SR::put4(sh, l32, col, hv[0], hv[1], hv[2], hv[3]);
          SR::put4(sa, l32, col, av[0], av[1], av[2], av[3]);
          SR::put4(su, l32, col, uv[0], uv[1], uv[2], uv[3]);
        }
      const int fc = f0 + wn * CoreT::GW + SR::col_of() * 8;
#pragma unroll
      for (int it = 0; it < SR::NI; ++it) {
        const int r = SR::row_of(it);
        const int64_t row = prow0 + r;
        const uint4 vh = SR::get(sh, r, SR::col_of());
        const uint4 va = SR::get(sa, r, SR::col_of());
        const uint4 vu = SR::get(su, r, SR::col_of());
        if (row < rend) {
          *reinterpret_cast<uint4*>(a.C + row * a.ldc + fc) = vh;
          if (a.C2) {
            *reinterpret_cast<uint4*>(a.C2 + row * a.ldc2 + fc) = va;
            *reinterpret_cast<uint4*>(a.C2 + row * a.ldc2 + a.F + fc) = vu;
          }
        }
      }
    } else if constexpr (EPI == kEpiSwigluBwd) {
      using SR = StagedRowsF32<CoreT::WN * 4>;
      const int nc = n0 + wn * CoreT::WN + SR::col_of() * 8;
#pragma unroll
      for (int jj = 0; jj < CoreT::NB; ++jj)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int q = g * 4;
          SR::put4(ep, l32, jj * 32 + g * 8 + c4, core.acc[i][jj][q], core.acc[i][jj][q + 1], core.acc[i][jj][q + 2],
                   core.acc[i][jj][q + 3]);
        }
      // saved A and U of the rows this lane stores, loaded once this block's
      // accumulators are staged (their registers are free again; loaded
      // before the staging, they made the kernel spill), overlapping the
      // read-back of the staged dH
      uint4 xa[SR::NI], xu[SR::NI];
#pragma unroll
      for (int it = 0; it < SR::NI; ++it) {
        const int64_t row = prow0 + SR::row_of(it);
        xa[it] = xu[it] = make_uint4(0, 0, 0, 0);
        if (row < rend) {
          xa[it] = *reinterpret_cast<const uint4*>(a.AU + row * a.ldau + nc);
          xu[it] = *reinterpret_cast<const uint4*>(a.AU + row * a.ldau + a.F + nc);
        }
      }
#pragma unroll
      for (int it = 0; it < SR::NI; ++it) {
        const int r = SR::row_of(it);
        const int64_t row = prow0 + r;
        // dH at columns nc .. nc + 7; saved A in [0, F), U in [F, 2F)
        float dh[8], A8[8], U8[8], da[8], du[8];
        SR::get8(ep, r, SR::col_of(), dh);
        if (row >= rend) continue;
        unpack8(xa[it], A8);
        unpack8(xu[it], U8);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float sg = 1.0f / (1.0f + __expf(-A8[e]));
          da[e] = dh[e] * U8[e] * (sg + A8[e] * sg * (1.0f - sg));
          du[e] = dh[e] * A8[e] * sg;
        }
        *reinterpret_cast<uint4*>(a.C + row * a.ldc + nc) = pack8(da);
        *reinterpret_cast<uint4*>(a.C + row * a.ldc + a.F + nc) = pack8(du);
      }
    } else {
      using SR = StagedRows<CoreT::WN * 2>;
      const int nc = n0 + wn * CoreT::WN + SR::col_of() * 8;
#pragma unroll
      for (int jj = 0; jj < CoreT::NB; ++jj)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int q = g * 4;
          SR::put4(ep, l32, jj * 32 + g * 8 + c4, core.acc[i][jj][q], core.acc[i][jj][q + 1], core.acc[i][jj][q + 2],
                   core.acc[i][jj][q + 3]);
        }
#pragma unroll
      for (int it = 0; it < SR::NI; ++it) {
        const int r = SR::row_of(it);
        const int64_t row = prow0 + r;
        const uint4 v = SR::get(ep, r, SR::col_of());
        if (row < rend) *reinterpret_cast<uint4*>(a.C + row * a.ldc + nc) = v;
      }
    }
  }
}

// Tail split of the row GEMM (the last, partial round of tiles cut along
// K): the partial sums of a piece stay in the MFMA register layout, one
// workspace slot per workgroup, then per wave, then per float4 index with
// the 64 lanes consecutive, so every store and load moves a whole 1 KiB.
//
// The pieces of a tile may run on different XCDs, whose L2 caches are not
// coherent with each other. The partial sums are therefore stored and loaded
// with device-scope coherence (the SC1 cache-policy bit: the store writes
// through to memory, the load does not take a stale L2 line), and a store is
// complete once the wave's vector-memory counter has drained. No device-wide
// fence is needed: such a fence would write back and invalidate the whole
// L2 of the XCD, evicting the operand tiles that every other workgroup there
// is using.
#ifndef FM_TAIL_SPREAD
#define FM_TAIL_SPREAD 1
#endif
#ifndef FM_SPLIT_MAX
#define FM_SPLIT_MAX 4
#endif
#ifndef FM_SPLIT_MIN_K
#define FM_SPLIT_MIN_K 32
#endif
// Cut a small partial last round of 256-wide tiles along N (0: never).
#ifndef FM_NSPLIT
#define FM_NSPLIT 1
#endif
constexpr int kSplitMax = FM_SPLIT_MAX;    // pieces per tile at most (2..4)
constexpr int kSplitMinK = FM_SPLIT_MIN_K;  // k-steps a tile needs before it is split
#ifndef FM_SPLIT_REGION_KIB
#define FM_SPLIT_REGION_KIB 16
#endif
constexpr int kSplitRegionKiB = FM_SPLIT_REGION_KIB;  // LDS per wave for the pieces in flight
constexpr int kCoherentDevice = 16;  // cache policy of buffer accesses: SC1

template <class CoreT, int NW>
__device__ __forceinline__ uint32_t split_offset(int slot, int wave, int e) {
  constexpr int PER_WAVE = CoreT::MB * CoreT::NB * 4 * 64;  // float4 per wave
  return (uint32_t)((((uint32_t)slot * NW + wave) * PER_WAVE + (uint32_t)e * 64 + lane64()) * 16u);
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t split_rsrc(float* part, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(part, (short)0, (int)bytes, 0x00020000);
}

// One wavefront moves 64 x 16 bytes of the split workspace into LDS (lane l
// to lds_wave_base + 16 l), device-coherently.
__device__ __forceinline__ void split_dma16(__amdgpu_buffer_rsrc_t rs, uint32_t lds_wave_base, uint32_t voff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (__attribute__((address_space(3))) void*)(uintptr_t)lds_wave_base, 16,
                                           voff, 0, 0, kCoherentDevice);
}

template <class CoreT, int NW>
__device__ __forceinline__ void split_store(__amdgpu_buffer_rsrc_t rs, int slot, int wave, const CoreT& core) {
#pragma unroll
  for (int i = 0; i < CoreT::MB; ++i)
#pragma unroll
    for (int j = 0; j < CoreT::NB; ++j)
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        i32x4 v;
        v.x = __float_as_int(core.acc[i][j][4 * c]);
        v.y = __float_as_int(core.acc[i][j][4 * c + 1]);
        v.z = __float_as_int(core.acc[i][j][4 * c + 2]);
        v.w = __float_as_int(core.acc[i][j][4 * c + 3]);
        __builtin_amdgcn_raw_buffer_store_b128(v, rs, split_offset<CoreT, NW>(slot, wave, (i * CoreT::NB + j) * 4 + c),
                                               0, kCoherentDevice);
      }
}

// acc = piece 0 + piece 1 + ... + piece SPLIT-1, added in this order for
// every element, all read back from the workspace (this workgroup's own
// piece included), so the result does not depend on which piece arrived
// last. The pieces travel workspace -> LDS by asynchronous loads that need
// no registers (up to 16 KiB per wave in flight, in the wave's own part of
// the free operand ring), then LDS -> registers for the additions. (Taking
// the own piece from the registers instead saves one read but makes the
// compiler spill the accumulators.) `rs` covers the tile's SPLIT slots;
// `wl` is the wave's LDS region.
template <int NW, int SPLIT, class CoreT>
__device__ __forceinline__ void split_sum(__amdgpu_buffer_rsrc_t rs, int wave, char* wl, CoreT& core) {
  constexpr int NE = CoreT::MB * CoreT::NB * 4;  // float4 groups per lane
  constexpr int GR = kSplitRegionKiB / SPLIT;    // groups per round
  const uint32_t wbase = lds_addr(wl);
  static_for<0, (NE + GR - 1) / GR>([&](auto rc) {
    constexpr int e0 = decltype(rc)::value * GR;
    constexpr int ne = NE - e0 < GR ? NE - e0 : GR;
#pragma unroll
    for (int g = 0; g < ne; ++g)
#pragma unroll
      for (int pc = 0; pc < SPLIT; ++pc)
        split_dma16(rs, wbase + (pc * GR + g) * 1024, split_offset<CoreT, NW>(pc, wave, e0 + g));
    wait_vm<0>();  // this wave's loads have landed in its LDS region
#pragma unroll
    for (int g = 0; g < ne; ++g) {
      const int e = e0 + g, c = e % 4, j = (e / 4) % CoreT::NB, i = e / 4 / CoreT::NB;
      float4 t = *reinterpret_cast<const float4*>(wl + g * 1024 + lane64() * 16);
#pragma unroll
      for (int pc = 1; pc < SPLIT; ++pc) {
        const float4 x = *reinterpret_cast<const float4*>(wl + (pc * GR + g) * 1024 + lane64() * 16);
        t.x += x.x;
        t.y += x.y;
        t.z += x.z;
        t.w += x.w;
      }
      core.acc[i][j][4 * c] = t.x;
      core.acc[i][j][4 * c + 1] = t.y;
      core.acc[i][j][4 * c + 2] = t.z;
      core.acc[i][j][4 * c + 3] = t.w;
    }
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): LDS reads done before the region is refilled
  });
}

template <int BM, int BN, int BK, int NS, int WGM, int WGN, bool B_KMAJ, int EPI>
__global__ __launch_bounds__(64 * WGM * WGN) void gemm_rows_kernel(RowsArgs a) {
  constexpr bool SW = (EPI == kEpiSwigluFwd);
  constexpr int NW = WGM * WGN;
  using CoreT = Core<BM, BN, WGM, WGN, SW>;
  using AT = KTile<BM, BK, NW>;
  using BT = typename std::conditional<B_KMAJ, KTile<BN, BK, NW>, MTile<BN, BK, NW>>::type;
  constexpr int STAGE = AT::BYTES + BT::BYTES;
  __shared__ __attribute__((aligned(1024))) char lds[NS * STAGE];
  __shared__ int s_mt[FOREMOE_MAX_SLOTS + 1];
  __shared__ int s_tmp[16];
  __shared__ int s_last;

  build_slot_tiles<BM>(a.slot_offset, a.S, a.n_cap, s_mt, s_tmp);
  const int n_tiles = a.N / BN;
  const int total = s_mt[a.S] * n_tiles;
  const int wave = wave_id();
  const int wm = wave / WGN, wn = wave % WGN;
  const int KT = a.K / BK;
  const uint32_t lds0 = lds_addr(lds);

  CoreT core;
  const typename CoreT::template Offsets<AT, BT, BK> offs(wm, wn);

  // Whole rounds of G tiles, one tile per workgroup per round. When the last
  // round is partial (r < G tiles), its tiles may be cut into `halves`
  // along N and, with a workspace, each (half) tile into `split` pieces
  // along K, so that r * halves * split workgroups share it instead of r.
  // The halves and pieces of one tile run on workgroups of one XCD.
  const int G = gridDim.x;
  const int v = xcd_virtual_id();
  const int r = total % G;
  int split = 1;
  // With 256-wide tiles, a partial last round of at most 7/16 G tiles is
  // first cut along N: each tile becomes two half-width tiles on two
  // workgroups, with no partial sums (measured faster than cutting the same
  // round along K). The K split then applies to the (half) tiles.
  int halves = 1;
  if constexpr (BN == 256 && FM_NSPLIT) halves = (r > 0 && 16 * r <= 7 * G) ? 2 : 1;
  if (a.sk_part && r > 0 && KT >= kSplitMinK) {
    // as many pieces as keep at most 7/8 of the workgroups busy, so that
    // the round is also spread over the XCDs (below); a split that fills
    // the GPU measured slower than the unsplit round spread out
    split = (7 * G / 8) / (r * halves);
    split = split < kSplitMax ? split : kSplitMax;
    if (split < 2) split = 1;
  }
  const int full = total - r;  // tiles of the whole rounds
  // One output tile, k-steps [kb, kb + nk). With pieces > 1 this is piece q
  // of a (half) tile cut along K: the partial sums go to the workspace and
  // the last piece to arrive adds all pieces in piece order and writes the
  // (half) tile. half_c = std::true_type: only columns
  // [h BN / 2, (h + 1) BN / 2) of tile t, each wave owning WM x WN / 2 (a
  // tile of the last round cut along N, below).
  auto run_tile = [&](auto half_c, int t, int h, int kb, int nk, int q, int pieces, int slot) {
    constexpr bool HALF = decltype(half_c)::value;
    constexpr int BNX = HALF ? BN / 2 : BN;
    using CoreX = typename std::conditional<HALF, Core<BM, BNX, WGM, WGN, SW>, CoreT>::type;
    using BTX = typename std::conditional<B_KMAJ, KTile<BNX, BK, NW>, MTile<BNX, BK, NW>>::type;
    constexpr int STAGEX = AT::BYTES + BTX::BYTES;
    const int mtg = t / n_tiles, nt = t % n_tiles;
    int lo = 0, hi = a.S - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (s_mt[mid] <= mtg) lo = mid;
      else hi = mid - 1;
    }
    const int j = __builtin_amdgcn_readfirstlane(lo);
    int64_t rbeg = a.slot_offset[j], rend = a.slot_offset[j + 1];
    rbeg = rbeg < 0 ? 0 : (rbeg > a.n_cap ? a.n_cap : rbeg);
    rend = rend < 0 ? 0 : (rend > a.n_cap ? a.n_cap : rend);
    const int mrel = (mtg - s_mt[j]) * BM;  // first tile row relative to the slot
    const int64_t m0 = rbeg + mrel;
    const int w = a.slot_widx[j];
    if (w < 0 || w >= a.W) return;  // invalid weight index: rows left unwritten (every piece skips)
    const int n0 = nt * BN + h * BNX;          // first output column of the tile grid
    const int f0 = nt * (BN / 2) + h * (BNX / 2);  // SwiGLU: first H column

    // operand A: the slot's rows only (rows past the slot read as zero);
    // operand B: weight matrix w. Lane offsets are fixed for the tile; each
    // stage moves the start of the buffer resource to its first k, so the
    // range check still ends at the slot's last row.
    const uint32_t lda2 = (uint32_t)(a.lda * 2), ldb2 = (uint32_t)(a.ldb * 2);
    const uint16_t* abase = a.A + rbeg * a.lda;
    const uint32_t abytes = (uint32_t)((rend - rbeg) * a.lda * 2);
    const uint16_t* bbase = a.B + (int64_t)w * a.wstride;
    const uint32_t bbytes = (uint32_t)(a.wstride * 2);
    auto arow = [&](int r) -> uint32_t { return (uint32_t)(mrel + r) * lda2; };
    auto brow = [&](int r) -> uint32_t {
      if constexpr (B_KMAJ) {
        int wr;
        if constexpr (SW) wr = r < BNX / 2 ? f0 + r : a.F + f0 + (r - BNX / 2);
        else wr = n0 + r;
        return (uint32_t)wr * ldb2;
      } else {
        // K-major weights: element (n, k) at (k * ldb + n) * 2
        return (uint32_t)r * ldb2 + (uint32_t)n0 * 2u;
      }
    };
    const uint32_t va0 = AT::voff(arow, 0), vb0 = BTX::voff(brow, 0);
    uint32_t sa_[AT::PER_WAVE], sb_[BTX::PER_WAVE];
#pragma unroll
    for (int i = 0; i < AT::PER_WAVE; ++i) sa_[i] = __builtin_amdgcn_readfirstlane(AT::voff(arow, i) - va0);
#pragma unroll
    for (int i = 0; i < BTX::PER_WAVE; ++i) sb_[i] = __builtin_amdgcn_readfirstlane(BTX::voff(brow, i) - vb0);
    auto issue = [&](int kt, int p) {
      // stages past the last load nothing (zero-size resources)
      const bool live = kt < nk;
      const uint32_t sa = lds0 + (uint32_t)((kt % NS) * STAGEX);
      const uint32_t k0 = live ? (uint32_t)((kb + kt) * BK) : 0u;
      if (p < AT::PER_WAVE) {
        AT::issue_s(buf_rsrc(abase + k0, live ? abytes - 2u * k0 : 0u), sa, va0, sa_[p], p);
      } else if constexpr (B_KMAJ) {
        BTX::issue_s(buf_rsrc(bbase + k0, live ? bbytes - 2u * k0 : 0u), sa + AT::BYTES, vb0, sb_[p - AT::PER_WAVE],
                     p - AT::PER_WAVE);
      } else {
        BTX::issue_s(buf_rsrc(bbase + (int64_t)k0 * a.ldb, live ? bbytes - k0 * ldb2 : 0u), sa + AT::BYTES, vb0,
                     sb_[p - AT::PER_WAVE], p - AT::PER_WAVE);
      }
    };

    // After the k-loop: a K piece stores its partial sums and the last piece
    // of its tile to arrive adds all pieces in piece order; then the
    // epilogue. cr is the full or the half-width core.
    auto finish_tile = [&](auto& cr) {
      using C = typename std::remove_reference<decltype(cr)>::type;
      constexpr int BNC = C::WN * WGN;  // output columns this core covers
      if (pieces > 1) {
        // piece q' of this (half) tile is computed by the workgroup with
        // slot slot - q + q'; each keeps its partial sums in its own
        // workspace slot
        const __amdgpu_buffer_rsrc_t rs = split_rsrc(a.sk_part, (uint32_t)G * (BM * BN * 4));
        split_store<C, NW>(rs, slot, wave, cr);
        wait_vm<0>();  // this wave's partial sums have reached memory
        __syncthreads();
        const int cidx = (t - full) * (BN / BNC) + h;  // arrival counter of this (half) tile
        if (threadIdx.x == 0) s_last = atomicAdd(&a.sk_count[cidx], 1u) == (unsigned)(pieces - 1);
        __syncthreads();
        if (!s_last) return;
        // the tile's pieces: slots slot - q .. slot - q + pieces - 1
        {
          static_assert(NW * kSplitRegionKiB * 1024 <= NS * STAGE, "split pieces must fit in the ring");
          const __amdgpu_buffer_rsrc_t ts =
              split_rsrc(a.sk_part + (size_t)(slot - q) * (BM * BNC), (uint32_t)pieces * (BM * BNC * 4));
          char* wl = lds + wave * (kSplitRegionKiB * 1024);
          if (pieces == 2) split_sum<NW, 2>(ts, wave, wl, cr);
          else if (pieces == 3) split_sum<NW, 3>(ts, wave, wl, cr);
          else split_sum<NW, 4>(ts, wave, wl, cr);
        }
        if (threadIdx.x == 0) atomicExch(&a.sk_count[cidx], 0u);  // ready for the next call
      }
      static_assert(NW * EpiBytes<C, EPI>::PER_WAVE <= NS * STAGE, "epilogue staging must fit in the ring");
      __syncthreads();  // every wave is done reading the ring: it now stages the epilogue
      rows_epilogue<C, EPI>(a, cr, lds + wave * EpiBytes<C, EPI>::PER_WAVE, m0 + wm * C::WM, rend, n0, f0, wn);
      __syncthreads();  // staging reads done before the next tile's loads overwrite the ring
    };

    if constexpr (HALF) {
      static_assert(STAGEX <= STAGE, "the half-width ring fits in the ring");
      CoreX hc;
      const typename CoreX::template Offsets<AT, BTX, BK> ox(wm, wn);
      hc.zero();
      pipelined_k_loop<CoreX, AT, BTX, BK, NS, SW ? FM_FRAG_DIST_FWD : FM_FRAG_DIST>(hc, lds, nk, ox, issue);
      finish_tile(hc);
    } else {
      core.zero();
      pipelined_k_loop<CoreT, AT, BT, BK, NS, SW ? FM_FRAG_DIST_FWD : FM_FRAG_DIST>(core, lds, nk, offs, issue);
      finish_tile(core);
    }
  };

  // Whole rounds take the XCD-grouped ids. A partial last round that keeps
  // at most 7/8 of the workgroups busy is spread over all eight XCDs
  // instead, in blocks: XCD x takes tiles [x * tpx, (x + 1) * tpx), so that
  // neighbouring tiles (which share operand rows or weights) still share an
  // L2, with the halves and pieces of a tile on consecutive workgroups of
  // that XCD. The XCDs share only memory, so such a round runs faster on eight
  // partly busy XCDs than on fewer full ones.
  for (int t = v; t < full; t += G) run_tile(std::false_type{}, t, 0, 0, KT, 0, 1, v);
  const int per = halves * split;  // workgroups per tile of the last round
  const int busy = r * per;
  int u = v;
  if (FM_TAIL_SPREAD && G % 8 == 0 && 8 * busy <= 7 * G) {
    const int b = blockIdx.x, tpx = (r + 7) / 8;  // tiles per XCD
    if (tpx * per <= G / 8) {
      const int x = b % 8, c = b / 8, j = c / per, i = x * tpx + j;
      u = (j < tpx && i < r) ? i * per + c % per : busy;  // busy: idle workgroup
    }
  }
  if (u < busy) {
    // unit u: tile full + u / per, half (u % per) / split, K piece u % split
    const int q = u % split;
    const int kb = q * KT / split, ke = (q + 1) * KT / split;
    if constexpr (BN == 256 && FM_NSPLIT) {
      if (halves == 2) {
        run_tile(std::true_type{}, full + u / per, (u % per) / split, kb, ke - kb, q, split, u);
        return;
      }
    }
    run_tile(std::false_type{}, full + u / split, 0, kb, ke - kb, q, split, u);
  }
}

// ---------------------------------------------------------------------------
// Weight gradient: dW[g] (M x N, fp32) += sum over the rows of every slot
// with gradient index g of A[row, :]^T B[row, :].
//
// Work split: the row sequence of a group (the concatenated row ranges of
// its slots, in slot order) is cut into chunks of CH rows when the caller's
// workspace allows, so that one hot expert spreads over many CUs. Chunk 0 of
// a group adds its result straight into dW; chunks 1.. write fp32 partial
// tiles to the workspace, and wgrad_reduce_kernel (launched next on the same
// stream) adds them in chunk order. Every output element therefore has one
// fixed summation order: deterministic, no atomics on floats.
// ---------------------------------------------------------------------------
// One micro-step's operands of a weight-gradient call: rows [0, n_cap) of A
// and B, and its slot table.
struct WgradStep {
  const uint16_t* A;  // [n_cap, M]
  const uint16_t* B;  // [n_cap, N]
  const int32_t* slot_offset;
  const int32_t* slot_gidx;
  int S;
  int vbase;  // first virtual slot of this step (prefix of S over the steps before)
  int64_t n_cap;
};

struct WgradArgs {
  WgradStep step[FOREMOE_MAX_WGRAD_STEPS];
  int n_steps;
  int V;  // virtual slots: every step's slots, steps in order
  int64_t lda, ldb;
  int M, N;
  int G;
  float* C;  // dW[g] at C + g * gstride, row-major [M, N]
  int64_t ldc;
  int64_t gstride;
  float* part;  // partial tiles [p_max][BM * BN]
  int p_max;
  // with partial tiles: the plan the reduce kernel needs, written by
  // workgroup 0 of the main kernel: {groups with rows, chunk rows, then per
  // ordered group: gradient index, rows, first partial tile}
  int* plan_out;
  // work counters {next item, finished workgroups} (zero on entry, zeroed
  // again by the last workgroup), or NULL for a static item order
  unsigned* sched;
  // output tiles of this call: tile index t of a group's dW (row-major over
  // the BM x BN tiles) with t % tparts == tpart
  int tpart, tparts;
};

// Tiles of one group's dW that a call computes, and the index of the i-th.
__device__ __forceinline__ int wgrad_call_tiles(const WgradArgs& a, int BM, int BN) {
  return ((a.M / BM) * (a.N / BN) - a.tpart + a.tparts - 1) / a.tparts;
}
__device__ __forceinline__ int wgrad_tile(const WgradArgs& a, int i) { return a.tpart + i * a.tparts; }

// The row sequence of gradient group g is the rows of every virtual slot v
// (step m's slot j, v = vbase_m + j) with gradient index g, in v order: the
// micro-steps in order, each one's slots in order.
struct WgradPlan {
  int beg[FOREMOE_MAX_SLOTS];        // clamped row range [beg, end) of virtual slot v in its step's rows
  int end[FOREMOE_MAX_SLOTS];
  int gs[FOREMOE_MAX_SLOTS];         // step << 16 | gradient index, -1 for empty/invalid slots
  int rows[FOREMOE_MAX_SLOTS];       // rows per group
  int order[FOREMOE_MAX_SLOTS];      // groups by descending rows
  int ibase[FOREMOE_MAX_SLOTS + 1];  // work-item prefix over ordered groups
  int pbase[FOREMOE_MAX_SLOTS + 1];  // partial-tile prefix over ordered groups
  const uint16_t* A[FOREMOE_MAX_WGRAD_STEPS];  // operands of each step
  const uint16_t* B[FOREMOE_MAX_WGRAD_STEPS];
  int nne;                           // non-empty groups
  int ch;                            // chunk rows (INT_MAX: no split)
  __device__ __forceinline__ int gidx(int v) const { return gs[v] < 0 ? -1 : (gs[v] & 0xFFFF); }
  __device__ __forceinline__ int step(int v) const { return gs[v] >> 16; }
};

template <int BM, int BN, int BK>
__device__ void build_wgrad_plan(const WgradArgs& a, WgradPlan& P) {
  const int tid = threadIdx.x;
  const int G = a.G, V = a.V;
  const int tpg = wgrad_call_tiles(a, BM, BN);
  const int nt = blockDim.x;
  if (tid == 0) P.nne = 0;
  // the step table into LDS with compile-time indices (a kernel argument
  // indexed at run time would be copied to scratch)
#pragma unroll
  for (int m = 0; m < FOREMOE_MAX_WGRAD_STEPS; ++m) {
    if (tid == m && m < a.n_steps) {
      P.A[m] = a.step[m].A;
      P.B[m] = a.step[m].B;
    }
  }
  for (int g = tid; g < G; g += nt) P.rows[g] = 0;
  for (int v = tid; v < V; v += nt) {
    int m = 0;
#pragma unroll
    for (int q = 1; q < FOREMOE_MAX_WGRAD_STEPS; ++q)
      if (q < a.n_steps && v >= a.step[q].vbase) m = q;
    const int32_t* off = nullptr;
    const int32_t* gi = nullptr;
    int64_t n_cap = 0;
    int j = 0;
#pragma unroll
    for (int q = 0; q < FOREMOE_MAX_WGRAD_STEPS; ++q)
      if (q == m) {
        off = a.step[q].slot_offset;
        gi = a.step[q].slot_gidx;
        n_cap = a.step[q].n_cap;
        j = v - a.step[q].vbase;
      }
    int64_t lo = off[j], hi = off[j + 1];
    lo = lo < 0 ? 0 : (lo > n_cap ? n_cap : lo);
    hi = hi < 0 ? 0 : (hi > n_cap ? n_cap : hi);
    const int g = gi[j];
    const bool ok = g >= 0 && g < G && hi > lo;
    P.beg[v] = (int)lo;
    P.end[v] = ok ? (int)hi : (int)lo;
    P.gs[v] = ok ? (m << 16 | g) : -1;
  }
  __syncthreads();
  for (int v = tid; v < V; v += nt)
    if (P.gs[v] >= 0) atomicAdd(&P.rows[P.gidx(v)], P.end[v] - P.beg[v]);
  __syncthreads();
  for (int g = tid; g < G; g += nt) {
    const int rg = P.rows[g];
    if (rg <= 0) continue;
    int rank = 0;
    for (int h = 0; h < G; ++h) {
      const int rh = P.rows[h];
      rank += (rh > rg) || (rh == rg && h < g);
    }
    P.order[rank] = g;
    atomicAdd(&P.nne, 1);
  }
  __syncthreads();
  if (tid == 0) {
    long long total = 0;
    for (int i = 0; i < P.nne; ++i) total += P.rows[P.order[i]];
    int ch = INT_MAX;
    if (a.p_max > 0 && total > 0) {
      long long c = (total * tpg + a.p_max - 1) / a.p_max;
      c = (c + BK - 1) / BK * BK;
      if (c < BK) c = BK;
      ch = c > INT_MAX ? INT_MAX : (int)c;
    }
    P.ch = ch;
    int ib = 0, pb = 0;
    for (int i = 0; i < P.nne; ++i) {
      const int rg = P.rows[P.order[i]];
      const int cg = ch == INT_MAX ? 1 : (rg + ch - 1) / ch;
      P.ibase[i] = ib;
      P.pbase[i] = pb;
      ib += cg * tpg;
      pb += (cg - 1) * tpg;
    }
    P.ibase[P.nne] = ib;
    P.pbase[P.nne] = pb;
  }
  __syncthreads();
}

// Walks the k-tiles of one chunk [s0, s1) of a group's row sequence: each
// k-tile lies inside one virtual slot's row range [lo, hi).
struct KCursor {
  int j, pos, lo, hi, k;  // virtual slot, sequence position of slot start, segment rows, tile start
  bool done;
  const uint16_t* pa;  // operands of slot j's micro-step (wave-uniform: scalar registers)
  const uint16_t* pb;
};

__device__ __forceinline__ const uint16_t* uniform_ptr(const uint16_t* p) {
  const uint64_t v = (uint64_t)p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return (const uint16_t*)(((uint64_t)hi << 32) | lo);
}

__device__ __forceinline__ void cursor_next_slot(const WgradPlan& P, int V, int g, int s1, KCursor& c) {
  int j = c.j, pos = c.pos;
  for (;;) {
    if (j >= 0 && P.gidx(j) == g) pos += P.end[j] - P.beg[j];
    ++j;
    if (j >= V || pos >= s1) {
      c.done = true;
      return;
    }
    if (P.gidx(j) == g) break;
  }
  c.j = j;
  c.pos = pos;
  c.lo = P.beg[j];
  const int n = P.end[j] - P.beg[j];
  c.hi = P.beg[j] + (n < s1 - pos ? n : s1 - pos);
  c.k = c.lo;
  c.pa = uniform_ptr(P.A[P.step(j)]);
  c.pb = uniform_ptr(P.B[P.step(j)]);
}

__device__ __forceinline__ KCursor cursor_begin(const WgradPlan& P, int V, int g, int s0, int s1) {
  KCursor c;
  c.done = false;
  int pos = 0;
  for (int j = 0; j < V; ++j) {
    if (P.gidx(j) != g) continue;
    const int n = P.end[j] - P.beg[j];
    if (pos + n > s0) {
      c.j = j;
      c.pos = pos;
      c.lo = P.beg[j] + (s0 - pos);
      c.hi = P.beg[j] + (n < s1 - pos ? n : s1 - pos);
      c.k = c.lo;
      c.pa = uniform_ptr(P.A[P.step(j)]);
      c.pb = uniform_ptr(P.B[P.step(j)]);
      return c;
    }
    pos += n;
  }
  c.done = true;
  c.pa = uniform_ptr(P.A[0]);
  c.pb = uniform_ptr(P.B[0]);
  return c;
}

template <int BK>
__device__ __forceinline__ void cursor_advance(const WgradPlan& P, int V, int g, int s1, KCursor& c) {
  c.k += BK;
  if (c.k >= c.hi) cursor_next_slot(P, V, g, s1, c);
}

template <int BM, int BN, int BK, int NS, int WGM, int WGN>
__global__ __launch_bounds__(64 * WGM * WGN) void gemm_wgrad_kernel(WgradArgs a) {
  constexpr int NW = WGM * WGN;
  using CoreT = Core<BM, BN, WGM, WGN, false>;
  using AT = MTile<BM, BK, NW>;
  using BT = MTile<BN, BK, NW>;
  constexpr int STAGE = AT::BYTES + BT::BYTES;
  __shared__ __attribute__((aligned(1024))) char lds[NS * STAGE];
  __shared__ WgradPlan P;

  build_wgrad_plan<BM, BN, BK>(a, P);
  if (a.plan_out && blockIdx.x == 0) {
    if (threadIdx.x == 0) {
      a.plan_out[0] = P.nne;
      a.plan_out[1] = P.ch;
    }
    for (int i = threadIdx.x; i < P.nne; i += blockDim.x) {
      a.plan_out[2 + 3 * i] = P.order[i];
      a.plan_out[3 + 3 * i] = P.rows[P.order[i]];
      a.plan_out[4 + 3 * i] = P.pbase[i];
    }
  }
  const int V = a.V;
  const int nt_n = a.N / BN, tpg = wgrad_call_tiles(a, BM, BN);
  const int total = P.ibase[P.nne];
  const int lane = lane64(), wave = wave_id();
  const int wm = wave / WGN, wn = wave % WGN;
  const uint32_t lds0 = lds_addr(lds);
  const uint32_t lda2 = (uint32_t)(a.lda * 2), ldb2 = (uint32_t)(a.ldb * 2);
  CoreT core;
  const typename CoreT::template Offsets<AT, BT, BK> offs(wm, wn);

  // Items (output tile x row chunk) come in descending group size. With
  // work counters each workgroup takes the next item when it is free, which
  // balances the very uneven item sizes; without, a fixed stride (XCD-aware).
  __shared__ int s_item;
  auto next_item = [&](int prev) -> int {
    if (!a.sched) return prev < 0 ? xcd_virtual_id() : prev + (int)gridDim.x;
    if (threadIdx.x == 0) s_item = (int)atomicAdd(&a.sched[0], 1u);
    __syncthreads();
    return s_item;
  };
  for (int t = next_item(-1); t < total; t = next_item(t)) {
    int lo = 0, hi = P.nne - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (P.ibase[mid] <= t) lo = mid;
      else hi = mid - 1;
    }
    const int gi = __builtin_amdgcn_readfirstlane(lo);
    const int g = P.order[gi];
    const int local = t - P.ibase[gi];
    const int c = local / tpg, tile_l = local % tpg, tile = wgrad_tile(a, tile_l);
    const int m0 = (tile / nt_n) * BM, n0 = (tile % nt_n) * BN;
    const int rg = P.rows[g];
    const int s0 = P.ch == INT_MAX ? 0 : c * P.ch;
    const int s1 = P.ch == INT_MAX ? rg : (s0 + P.ch < rg ? s0 + P.ch : rg);

    // number of k-tiles of this chunk (each k-tile stays inside one slot)
    int KT = 0;
    for (KCursor cc = cursor_begin(P, V, g, s0, s1); !cc.done; cursor_next_slot(P, V, g, s1, cc))
      KT += (cc.hi - cc.lo + BK - 1) / BK;
    KCursor ic = cursor_begin(P, V, g, s0, s1);
    auto koa = [&](int k) -> uint32_t { return (uint32_t)k * lda2 + (uint32_t)m0 * 2u; };
    auto kob = [&](int k) -> uint32_t { return (uint32_t)k * ldb2 + (uint32_t)n0 * 2u; };
    const uint32_t va0 = AT::voff(koa, 0), vb0 = BT::voff(kob, 0);
    uint32_t sa_[AT::PER_WAVE], sb_[BT::PER_WAVE];
#pragma unroll
    for (int i = 0; i < AT::PER_WAVE; ++i) sa_[i] = __builtin_amdgcn_readfirstlane(AT::voff(koa, i) - va0);
#pragma unroll
    for (int i = 0; i < BT::PER_WAVE; ++i) sb_[i] = __builtin_amdgcn_readfirstlane(BT::voff(kob, i) - vb0);
    auto issue = [&](int kt, int p) {
      // the loads of one k-tile are issued in order p = 0 .. PER-1, k-tiles
      // in order: load the cursor's k-tile, advance after its last load. The
      // resource starts at the k-tile's first row and ends at the segment's
      // last, so rows past the segment read as zero; once the cursor is
      // done, the stages past the last load nothing.
      const bool live = !ic.done;
      const uint32_t sa = lds0 + (uint32_t)((kt % NS) * STAGE);
      const int k = live ? ic.k : 0;
      const uint32_t nrow = live ? (uint32_t)(ic.hi - ic.k) : 0u;
      if (p < AT::PER_WAVE) {
        AT::issue_s(buf_rsrc(ic.pa + (int64_t)k * a.lda, nrow * lda2), sa, va0, sa_[p], p);
      } else {
        BT::issue_s(buf_rsrc(ic.pb + (int64_t)k * a.ldb, nrow * ldb2), sa + AT::BYTES, vb0, sb_[p - AT::PER_WAVE],
                    p - AT::PER_WAVE);
      }
      if (p == AT::PER_WAVE + BT::PER_WAVE - 1 && live) cursor_advance<BK>(P, V, g, s1, ic);
    };

    core.zero();
    pipelined_k_loop<CoreT, AT, BT, BK, NS>(core, lds, KT, offs, issue);
    __syncthreads();

    const int l32 = lane & 31, c4 = (lane >> 5) * 4;
    if (c == 0) {
      // dW += acc. The current dW values of this wave's output are brought
      // into LDS with asynchronous buffer loads (two 32-row blocks at a time,
      // all loads in flight together; each wave uses its own LDS region, so
      // no barrier is needed), then added to the accumulators and stored.
      float* Cg = a.C + (int64_t)g * a.gstride;
      constexpr int RB = CoreT::WN * 4;  // bytes of one output row of this wave
      constexpr int CH = RB / 16;        // 16-byte chunks per row
      constexpr int REGION = 2 * 32 * RB;
      static_assert(NW * REGION <= NS * STAGE, "epilogue staging must fit the LDS stages");
      static_assert(CH >= 16 && (CH & (CH - 1)) == 0, "row chunks");
      const i32x4 rsc = buf_rsrc(Cg, (uint32_t)((int64_t)a.M * a.N * 4));
      char* wl = lds + wave * REGION;
      const int nb = n0 + wn * CoreT::WN;
#pragma unroll
      for (int ph = 0; ph < (CoreT::MB + 1) / 2; ++ph) {
#pragma unroll
        for (int ii = 0; ii < 2; ++ii) {
          const int i = ph * 2 + ii;
          if (i >= CoreT::MB) break;
          const int mb = m0 + wm * CoreT::WM + i * 32;
#pragma unroll
          for (int q = 0; q < 32 * RB / 1024; ++q) {
            const int r = q * (1024 / RB) + (lane * 16) / RB;
            const int pc = ((lane * 16) % RB) / 16;
            const int lc = pc ^ (r & (CH - 1));
            dma16(rsc, lds_addr(wl + ii * (32 * RB) + q * 1024),
                  (uint32_t)(((int64_t)(mb + r) * a.ldc + nb) * 4) + (uint32_t)lc * 16u);
          }
        }
        wait_vm<0>();
        // add the accumulators in place (LDS row r, chunk pc holds the
        // global chunk pc ^ (r % CH) of row r)...
#pragma unroll
        for (int ii = 0; ii < 2; ++ii) {
          const int i = ph * 2 + ii;
          if (i >= CoreT::MB) break;
#pragma unroll
          for (int jj = 0; jj < CoreT::NB; ++jj) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const int nl = jj * 32 + q * 8 + c4;
              const int pc = (nl / 4) ^ (l32 & (CH - 1));
              float4* lp = reinterpret_cast<float4*>(wl + ii * (32 * RB) + l32 * RB + pc * 16);
              float4 o = *lp;
              o.x += core.acc[i][jj][q * 4 + 0];
              o.y += core.acc[i][jj][q * 4 + 1];
              o.z += core.acc[i][jj][q * 4 + 2];
              o.w += core.acc[i][jj][q * 4 + 3];
              *lp = o;
            }
          }
        }
        __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): the sums are in LDS
        // ...then store them from the lanes that loaded them: each store
        // instruction writes whole row segments (full 128-byte lines)
#pragma unroll
        for (int ii = 0; ii < 2; ++ii) {
          const int i = ph * 2 + ii;
          if (i >= CoreT::MB) break;
          const int mb = m0 + wm * CoreT::WM + i * 32;
#pragma unroll
          for (int q = 0; q < 32 * RB / 1024; ++q) {
            const int r = q * (1024 / RB) + (lane * 16) / RB;
            const int pc = ((lane * 16) % RB) / 16;
            const int lc = pc ^ (r & (CH - 1));
            const float4 o = *reinterpret_cast<const float4*>(wl + ii * (32 * RB) + q * 1024 + lane * 16);
            *reinterpret_cast<float4*>(Cg + (int64_t)(mb + r) * a.ldc + nb + lc * 4) = o;
          }
        }
        __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): LDS reads done before the region is refilled
      }
    } else {
      float* Pt = a.part + (int64_t)(P.pbase[gi] + (c - 1) * tpg + tile_l) * (BM * BN);
#pragma unroll
      for (int i = 0; i < CoreT::MB; ++i) {
        const int m = wm * CoreT::WM + i * 32 + l32;
#pragma unroll
        for (int jj = 0; jj < CoreT::NB; ++jj) {
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int n = wn * CoreT::WN + jj * 32 + q * 8 + c4;
            *reinterpret_cast<float4*>(Pt + m * BN + n) =
                make_float4(core.acc[i][jj][q * 4 + 0], core.acc[i][jj][q * 4 + 1], core.acc[i][jj][q * 4 + 2],
                            core.acc[i][jj][q * 4 + 3]);
          }
        }
      }
    }
    __syncthreads();  // the epilogue's LDS staging is done before the next item's loads
  }
  if (a.sched && threadIdx.x == 0) {
    // each workgroup counts itself finished after its last take returned, so
    // the last one to finish can zero the counters for the next call
    if (atomicAdd(&a.sched[1], 1u) == gridDim.x - 1) {
      atomicExch(&a.sched[0], 0u);
      atomicExch(&a.sched[1], 0u);
    }
  }
}

// dW[g] tile += partials of chunks 1.. in chunk order. Each tile is cut into
// kReduceParts row bands, one workgroup per band, so that all CUs stream.
constexpr int kReduceParts = 16;

template <int BM, int BN, int BK>
__global__ __launch_bounds__(256) void wgrad_reduce_kernel(WgradArgs a) {
  // the main kernel's plan (its split groups come first: largest rows)
  const int* pl = a.plan_out;
  const int nne = pl[0], ch = pl[1];
  if (ch == INT_MAX) return;
  const int nt_n = a.N / BN, tpg = wgrad_call_tiles(a, BM, BN);
  int nsplit = 0;
  while (nsplit < nne && (pl[3 + 3 * nsplit] + ch - 1) / ch > 1) ++nsplit;
  const int total = nsplit * tpg * kReduceParts;
  constexpr int BAND = BM * BN / kReduceParts;  // elements per band
  constexpr int V = BAND / 1024 < 4 ? BAND / 1024 : 4;  // float4 per thread per pass
  static_assert(V >= 1 && BAND % (256 * 4 * V) == 0, "band split");
  for (int t = blockIdx.x; t < total; t += gridDim.x) {
    const int part = t % kReduceParts, tt = t / kReduceParts;
    const int gi = tt / tpg, tile_l = tt % tpg, tile = wgrad_tile(a, tile_l);
    const int g = pl[2 + 3 * gi];
    const int cg = (pl[3 + 3 * gi] + ch - 1) / ch;
    const int m0 = (tile / nt_n) * BM, n0 = (tile % nt_n) * BN;
    float* Cg = a.C + (int64_t)g * a.gstride;
    const float* P0 = a.part + (int64_t)(pl[4 + 3 * gi] + tile_l) * (BM * BN);
    const int64_t cstride = (int64_t)tpg * (BM * BN);
    for (int e0 = part * BAND + threadIdx.x * 4; e0 < (part + 1) * BAND; e0 += 256 * 4 * V) {
      float4 s[V];
#pragma unroll
      for (int v = 0; v < V; ++v) s[v] = *reinterpret_cast<const float4*>(P0 + e0 + v * 1024);
      for (int c = 2; c < cg; ++c) {
        float4 x[V];
#pragma unroll
        for (int v = 0; v < V; ++v) x[v] = *reinterpret_cast<const float4*>(P0 + (c - 1) * cstride + e0 + v * 1024);
#pragma unroll
        for (int v = 0; v < V; ++v) {
          s[v].x += x[v].x;
          s[v].y += x[v].y;
          s[v].z += x[v].z;
          s[v].w += x[v].w;
        }
      }
      float4 o[V];
#pragma unroll
      for (int v = 0; v < V; ++v) {
        const int e = e0 + v * 1024;
        o[v] = *reinterpret_cast<const float4*>(Cg + (int64_t)(m0 + e / BN) * a.ldc + n0 + e % BN);
      }
#pragma unroll
      for (int v = 0; v < V; ++v) {
        const int e = e0 + v * 1024;
        o[v].x += s[v].x;
        o[v].y += s[v].y;
        o[v].z += s[v].z;
        o[v].w += s[v].w;
        *reinterpret_cast<float4*>(Cg + (int64_t)(m0 + e / BN) * a.ldc + n0 + e % BN) = o[v];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// fp32 path: one thread per output element (small shapes).
// ---------------------------------------------------------------------------
__device__ __forceinline__ int find_slot(const int32_t* __restrict__ off, int S, int64_t row) {
  // last slot j with off[j] <= row (row < off[S] is guaranteed by the caller)
  int lo = 0, hi = S - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (off[mid] <= row) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

enum F32Op { kF32GateUpFwd = 0, kF32DownFwd = 1, kF32DownDgrad = 2, kF32GateUpDgrad = 3 };

template <int OP>
__global__ __launch_bounds__(256) void f32_rows_kernel(const float* __restrict__ A, const float* __restrict__ Wt,
                                                       const float* __restrict__ AU, int d, int F, int W,
                                                       const int32_t* __restrict__ off, const int32_t* __restrict__ widx,
                                                       int S, int64_t n_cap, float* __restrict__ C,
                                                       float* __restrict__ C2) {
  const int col = blockIdx.x * 16 + (threadIdx.x & 15);
  const int64_t row = (int64_t)blockIdx.y * 16 + (threadIdx.x >> 4);
  if (S <= 0) return;
  int64_t N = off[S];
  if (N > n_cap) N = n_cap;
  if (row >= N) return;
  const int ncols = (OP == kF32GateUpFwd || OP == kF32DownDgrad) ? F : d;
  if (col >= ncols) return;
  const int j = find_slot(off, S, row);
  const int w = widx[j];
  if (w < 0 || w >= W) return;
  if constexpr (OP == kF32GateUpFwd) {
    const float* x = A + row * d;
    const float* wg = Wt + (int64_t)w * 2 * F * d + (int64_t)col * d;
    const float* wu = wg + (int64_t)F * d;
    float av = 0.f, uv = 0.f;
    for (int k = 0; k < d; ++k) {
      av += x[k] * wg[k];
      uv += x[k] * wu[k];
    }
    C[row * F + col] = silu_f(av) * uv;
    if (C2) {
      C2[row * 2 * F + col] = av;
      C2[row * 2 * F + F + col] = uv;
    }
  } else if constexpr (OP == kF32DownFwd) {
    const float* h = A + row * F;
    const float* wd = Wt + (int64_t)w * d * F + (int64_t)col * F;
    float s = 0.f;
    for (int k = 0; k < F; ++k) s += h[k] * wd[k];
    C[row * d + col] = s;
  } else if constexpr (OP == kF32DownDgrad) {
    const float* dy = A + row * d;
    const float* wd = Wt + (int64_t)w * d * F + col;
    float dh = 0.f;
    for (int k = 0; k < d; ++k) dh += dy[k] * wd[(int64_t)k * F];
    const float av = AU[row * 2 * F + col], uv = AU[row * 2 * F + F + col];
    const float s = 1.0f / (1.0f + __expf(-av));
    C[row * 2 * F + col] = dh * uv * (s + av * s * (1.0f - s));
    C[row * 2 * F + F + col] = dh * av * s;
  } else {
    const float* dau = A + row * 2 * F;
    const float* wgu = Wt + (int64_t)w * 2 * F * d + col;
    float s = 0.f;
    for (int k = 0; k < 2 * F; ++k) s += dau[k] * wgu[(int64_t)k * d];
    C[row * d + col] = s;
  }
}

// dW[g][m][n] += sum over rows of slots with gidx g of A[row][m] * B[row][n]
__global__ __launch_bounds__(256) void f32_wgrad_kernel(const float* __restrict__ A, int lda, const float* __restrict__ B,
                                                        int ldb, int M, int N, const int32_t* __restrict__ off,
                                                        const int32_t* __restrict__ gidx, int S, int G, int64_t n_cap,
                                                        int part, int parts, float* __restrict__ C) {
  const int n = blockIdx.x * 16 + (threadIdx.x & 15);
  const int m = blockIdx.y * 16 + (threadIdx.x >> 4);
  const int g = blockIdx.z;
  if (n >= N || m >= M || m % parts != part) return;
  float s = 0.f;
  for (int j = 0; j < S; ++j) {
    if (gidx[j] != g) continue;
    int64_t lo = off[j], hi = off[j + 1];
    lo = lo < 0 ? 0 : (lo > n_cap ? n_cap : lo);
    hi = hi < 0 ? 0 : (hi > n_cap ? n_cap : hi);
    for (int64_t r = lo; r < hi; ++r) s += A[r * lda + m] * B[r * ldb + n];
  }
  C[((int64_t)g * M + m) * N + n] += s;
}

// ---------------------------------------------------------------------------
// Host launchers
// ---------------------------------------------------------------------------
int persistent_grid() { return num_cus(); }

// Row-GEMM workspace (optional): arrival counters of the split round, then
// one fp32 partial tile of up to 256 x 256 per workgroup of the grid.
constexpr size_t kRowsCountBytes = 4096;  // counters for up to 1024 tiles
constexpr size_t kRowsSlotBytes = (size_t)256 * 256 * 4;

size_t rows_workspace_bytes() { return kRowsCountBytes + (size_t)persistent_grid() * kRowsSlotBytes; }

// Row-grouped launches: 256-row tiles; 256-wide output tiles with 2 LDS
// stages of 64-deep K slices (128 KiB), or 128-wide with 3 stages (144 KiB).
// e0, e1: optional timing events set when the kernel starts and ends (they
// ride on the dispatch itself, so no event command sits in the stream).
template <int BN, bool KMAJ, int EPI>
void launch_rows(RowsArgs a, void* ws, hipStream_t st, hipEvent_t e0, hipEvent_t e1) {
  if (ws && persistent_grid() <= (int)(kRowsCountBytes / 4)) {
    a.sk_count = (unsigned*)ws;
    a.sk_part = (float*)((char*)ws + kRowsCountBytes);
  }
  if constexpr (BN == 256) {
    constexpr int WGM = FM_ROWS_WGM, WGN = FM_ROWS_WGN;
    hipExtLaunchKernelGGL(gemm_rows_kernel<256, 256, FM_ROWS_BK, FM_ROWS_NS, WGM, WGN, KMAJ, EPI>,
                          dim3(persistent_grid()), dim3(64 * WGM * WGN), 0, st, e0, e1, 0, a);
  } else {
    hipExtLaunchKernelGGL(gemm_rows_kernel<256, 128, 64, 3, 2, 2, KMAJ, EPI>, dim3(persistent_grid()), dim3(256), 0,
                          st, e0, e1, 0, a);
  }
}

// Weight-gradient workspace: a 256-byte header of work counters, then the
// partial-tile budget of the split (tiles of 256 x 256 fp32).
constexpr size_t kWgradHeaderBytes = 256;
constexpr size_t kWgradPlanBytes = 16384;  // the exported plan: 2 + 3 * FOREMOE_MAX_SLOTS ints
constexpr size_t kWgradPartialTiles = 256;
constexpr size_t kWgradWorkspaceBytes = kWgradHeaderBytes + kWgradPlanBytes + kWgradPartialTiles * 256 * 256 * 4;
static_assert((2 + 3 * FOREMOE_MAX_SLOTS) * 4 <= kWgradPlanBytes, "plan export region");

}  // namespace
}  // namespace foremoe

using namespace foremoe;

#define REQUIRE(cond, ...)                                      \
  do {                                                          \
    if (!(cond)) return set_error(FOREMOE_EINVAL, __VA_ARGS__); \
  } while (0)

static int check_ffn(const char* who, foremoe_dtype dtype, int32_t d, int32_t F, int32_t S, int64_t n_cap,
                     const int32_t* slot_offset) {
  REQUIRE(dtype == FOREMOE_F32 || dtype == FOREMOE_BF16, "%s: bad dtype", who);
  REQUIRE(d >= 1 && F >= 1, "%s: d and F must be positive", who);
  REQUIRE(S >= 0 && S <= FOREMOE_MAX_SLOTS, "%s: S=%d out of range", who, S);
  REQUIRE(n_cap >= 0 && n_cap < (int64_t)INT_MAX, "%s: n_cap out of range", who);
  REQUIRE(slot_offset, "%s: slot_offset is NULL", who);
  if (dtype == FOREMOE_BF16 && (d % 128 != 0 || F % 128 != 0))
    return set_error(FOREMOE_EUNSUPPORTED, "%s: bf16 needs d %% 128 == 0 and F %% 128 == 0 (d=%d, F=%d)", who, d, F);
  // 32-bit buffer offsets: (rows of one slot + one tile) * row bytes must fit
  if (dtype == FOREMOE_BF16 && (n_cap + 256) * (int64_t)(d > 2 * F ? d : 2 * F) * 2 >= ((int64_t)1 << 32))
    return set_error(FOREMOE_EUNSUPPORTED, "%s: (n_cap + 256) * row bytes must stay below 4 GiB", who);
  return FOREMOE_OK;
}

static int check_rows_ws(const char* who, const void* workspace, size_t ws_bytes) {
  if (!workspace) return FOREMOE_OK;
  REQUIRE(((uintptr_t)workspace & 255) == 0, "%s: workspace must be 256-byte aligned", who);
  REQUIRE(ws_bytes >= rows_workspace_bytes(), "%s: workspace of %zu bytes, %zu needed", who, ws_bytes,
          rows_workspace_bytes());
  return FOREMOE_OK;
}

// A timed call that launches nothing still sets its events, back to back on
// the stream, so that their elapsed time reads as zero.
static int no_launch(hipEvent_t e0, hipEvent_t e1, void* stream) {
  if (!e0 && !e1) return FOREMOE_OK;
  if (e0 && hipEventRecord(e0, (hipStream_t)stream) != hipSuccess)
    return set_error(FOREMOE_EHIP, "row GEMM: recording the start event failed");
  if (e1 && hipEventRecord(e1, (hipStream_t)stream) != hipSuccess)
    return set_error(FOREMOE_EHIP, "row GEMM: recording the stop event failed");
  return FOREMOE_OK;
}

static dim3 f32_grid(int cols, int64_t rows) {
  return dim3((unsigned)((cols + 15) / 16), (unsigned)((rows + 15) / 16 > 0 ? (rows + 15) / 16 : 1));
}

extern "C" {

static int ffn_gate_up_fwd_impl(const void* x_perm, foremoe_dtype dtype, int32_t d, int32_t F, int32_t S,
                            const int32_t* slot_offset, const int32_t* slot_widx, int32_t W, const void* w_gate_up,
                            int64_t n_cap, void* h, void* save_au, void* workspace, size_t ws_bytes, void* stream, hipEvent_t e0, hipEvent_t e1) {
  int rc = check_ffn("gate_up_fwd", dtype, d, F, S, n_cap, slot_offset);
  if (rc) return rc;
  rc = check_rows_ws("gate_up_fwd", workspace, ws_bytes);
  if (rc) return rc;
  if (S == 0 || n_cap == 0) return no_launch(e0, e1, stream);
  REQUIRE(x_perm && slot_widx && w_gate_up && h && W >= 1, "gate_up_fwd: NULL buffer or W < 1");
  hipStream_t st = (hipStream_t)stream;
  if (dtype == FOREMOE_BF16) {
    RowsArgs a{};
    a.A = (const uint16_t*)x_perm;
    a.lda = d;
    a.B = (const uint16_t*)w_gate_up;
    a.ldb = d;
    a.wstride = (int64_t)2 * F * d;
    a.W = W;
    a.K = d;
    a.N = 2 * F;
    a.F = F;
    a.slot_offset = slot_offset;
    a.slot_widx = slot_widx;
    a.S = S;
    a.n_cap = n_cap;
    a.C = (uint16_t*)h;
    a.ldc = F;
    a.C2 = (uint16_t*)save_au;
    a.ldc2 = 2 * (int64_t)F;
    launch_rows<256, true, kEpiSwigluFwd>(a, workspace, st, e0, e1);
  } else {
    hipExtLaunchKernelGGL(f32_rows_kernel<kF32GateUpFwd>, f32_grid(F, n_cap), dim3(256), 0, st, e0, e1, 0, (const float*)x_perm,
                       (const float*)w_gate_up, nullptr, d, F, W, slot_offset, slot_widx, S, n_cap, (float*)h,
                       (float*)save_au);
  }
  return check_launch("foremoe_ffn_gate_up_fwd");
}

static int ffn_down_fwd_impl(const void* h, foremoe_dtype dtype, int32_t d, int32_t F, int32_t S,
                         const int32_t* slot_offset, const int32_t* slot_widx, int32_t W, const void* w_down,
                         int64_t n_cap, void* y_perm, void* workspace, size_t ws_bytes, void* stream, hipEvent_t e0, hipEvent_t e1) {
  int rc = check_ffn("down_fwd", dtype, d, F, S, n_cap, slot_offset);
  if (rc) return rc;
  rc = check_rows_ws("down_fwd", workspace, ws_bytes);
  if (rc) return rc;
  if (S == 0 || n_cap == 0) return no_launch(e0, e1, stream);
  REQUIRE(h && slot_widx && w_down && y_perm && W >= 1, "down_fwd: NULL buffer or W < 1");
  hipStream_t st = (hipStream_t)stream;
  if (dtype == FOREMOE_BF16) {
    RowsArgs a{};
    a.A = (const uint16_t*)h;
    a.lda = F;
    a.B = (const uint16_t*)w_down;
    a.ldb = F;
    a.wstride = (int64_t)d * F;
    a.W = W;
    a.K = F;
    a.N = d;
    a.F = F;
    a.slot_offset = slot_offset;
    a.slot_widx = slot_widx;
    a.S = S;
    a.n_cap = n_cap;
    a.C = (uint16_t*)y_perm;
    a.ldc = d;
    if (d % 256 == 0) launch_rows<256, true, kEpiStore>(a, workspace, st, e0, e1);
    else launch_rows<128, true, kEpiStore>(a, workspace, st, e0, e1);
  } else {
    hipExtLaunchKernelGGL(f32_rows_kernel<kF32DownFwd>, f32_grid(d, n_cap), dim3(256), 0, st, e0, e1, 0, (const float*)h,
                       (const float*)w_down, nullptr, d, F, W, slot_offset, slot_widx, S, n_cap, (float*)y_perm,
                       nullptr);
  }
  return check_launch("foremoe_ffn_down_fwd");
}

int foremoe_grouped_ffn_fwd(const void* x_perm, foremoe_dtype dtype, int32_t d, int32_t F, int32_t S,
                            const int32_t* slot_offset, const int32_t* slot_widx, int32_t W, const void* w_gate_up,
                            const void* w_down, int64_t n_cap, void* h, void* y_perm, void* save_au, void* workspace, size_t ws_bytes, void* stream) {
  int rc = foremoe_ffn_gate_up_fwd(x_perm, dtype, d, F, S, slot_offset, slot_widx, W, w_gate_up, n_cap, h, save_au,
                                   workspace, ws_bytes, stream);
  if (rc) return rc;
  return foremoe_ffn_down_fwd(h, dtype, d, F, S, slot_offset, slot_widx, W, w_down, n_cap, y_perm, workspace, ws_bytes,
                              stream);
}

static int ffn_down_dgrad_impl(const void* dy_perm, const void* save_au, foremoe_dtype dtype, int32_t d, int32_t F,
                           int32_t S, const int32_t* slot_offset, const int32_t* slot_widx, int32_t W,
                           const void* w_down, int64_t n_cap, void* d_au, void* workspace, size_t ws_bytes, void* stream, hipEvent_t e0, hipEvent_t e1) {
  int rc = check_ffn("down_dgrad", dtype, d, F, S, n_cap, slot_offset);
  if (rc) return rc;
  rc = check_rows_ws("down_dgrad", workspace, ws_bytes);
  if (rc) return rc;
  if (S == 0 || n_cap == 0) return no_launch(e0, e1, stream);
  REQUIRE(dy_perm && save_au && slot_widx && w_down && d_au && W >= 1, "down_dgrad: NULL buffer or W < 1");
  hipStream_t st = (hipStream_t)stream;
  if (dtype == FOREMOE_BF16) {
    RowsArgs a{};
    a.A = (const uint16_t*)dy_perm;
    a.lda = d;
    a.B = (const uint16_t*)w_down;  // [d, F]: K-major for this product
    a.ldb = F;
    a.wstride = (int64_t)d * F;
    a.W = W;
    a.K = d;
    a.N = F;
    a.F = F;
    a.slot_offset = slot_offset;
    a.slot_widx = slot_widx;
    a.S = S;
    a.n_cap = n_cap;
    a.C = (uint16_t*)d_au;
    a.ldc = 2 * (int64_t)F;
    a.AU = (const uint16_t*)save_au;
    a.ldau = 2 * (int64_t)F;
    if (F % 256 == 0) launch_rows<256, false, kEpiSwigluBwd>(a, workspace, st, e0, e1);
    else launch_rows<128, false, kEpiSwigluBwd>(a, workspace, st, e0, e1);
  } else {
    hipExtLaunchKernelGGL(f32_rows_kernel<kF32DownDgrad>, f32_grid(F, n_cap), dim3(256), 0, st, e0, e1, 0, (const float*)dy_perm,
                       (const float*)w_down, (const float*)save_au, d, F, W, slot_offset, slot_widx, S, n_cap,
                       (float*)d_au, nullptr);
  }
  return check_launch("foremoe_ffn_down_dgrad");
}

static int ffn_gate_up_dgrad_impl(const void* d_au, foremoe_dtype dtype, int32_t d, int32_t F, int32_t S,
                              const int32_t* slot_offset, const int32_t* slot_widx, int32_t W, const void* w_gate_up,
                              int64_t n_cap, void* dx_perm, void* workspace, size_t ws_bytes, void* stream, hipEvent_t e0, hipEvent_t e1) {
  int rc = check_ffn("gate_up_dgrad", dtype, d, F, S, n_cap, slot_offset);
  if (rc) return rc;
  rc = check_rows_ws("gate_up_dgrad", workspace, ws_bytes);
  if (rc) return rc;
  if (S == 0 || n_cap == 0) return no_launch(e0, e1, stream);
  REQUIRE(d_au && slot_widx && w_gate_up && dx_perm && W >= 1, "gate_up_dgrad: NULL buffer or W < 1");
  hipStream_t st = (hipStream_t)stream;
  if (dtype == FOREMOE_BF16) {
    RowsArgs a{};
    a.A = (const uint16_t*)d_au;
    a.lda = 2 * (int64_t)F;
    a.B = (const uint16_t*)w_gate_up;  // [2F, d]: K-major for this product
    a.ldb = d;
    a.wstride = (int64_t)2 * F * d;
    a.W = W;
    a.K = 2 * F;
    a.N = d;
    a.F = F;
    a.slot_offset = slot_offset;
    a.slot_widx = slot_widx;
    a.S = S;
    a.n_cap = n_cap;
    a.C = (uint16_t*)dx_perm;
    a.ldc = d;
    if (d % 256 == 0) launch_rows<256, false, kEpiStore>(a, workspace, st, e0, e1);
    else launch_rows<128, false, kEpiStore>(a, workspace, st, e0, e1);
  } else {
    hipExtLaunchKernelGGL(f32_rows_kernel<kF32GateUpDgrad>, f32_grid(d, n_cap), dim3(256), 0, st, e0, e1, 0, (const float*)d_au,
                       (const float*)w_gate_up, nullptr, d, F, W, slot_offset, slot_widx, S, n_cap, (float*)dx_perm,
                       nullptr);
  }
  return check_launch("foremoe_ffn_gate_up_dgrad");
}

int foremoe_ffn_gate_up_fwd(const void* x_perm, foremoe_dtype dtype, int32_t d, int32_t F, int32_t S,
                            const int32_t* slot_offset, const int32_t* slot_widx, int32_t W, const void* w_gate_up,
                            int64_t n_cap, void* h, void* save_au, void* workspace, size_t ws_bytes, void* stream) {
  return ffn_gate_up_fwd_impl(x_perm, dtype, d, F, S, slot_offset, slot_widx, W, w_gate_up, n_cap, h, save_au,
                              workspace, ws_bytes, stream, nullptr, nullptr);
}

int foremoe_ffn_gate_up_fwd_timed(const void* x_perm, foremoe_dtype dtype, int32_t d, int32_t F, int32_t S,
                                  const int32_t* slot_offset, const int32_t* slot_widx, int32_t W,
                                  const void* w_gate_up, int64_t n_cap, void* h, void* save_au, void* workspace,
                                  size_t ws_bytes, void* stream, void* start_event, void* stop_event) {
  return ffn_gate_up_fwd_impl(x_perm, dtype, d, F, S, slot_offset, slot_widx, W, w_gate_up, n_cap, h, save_au,
                              workspace, ws_bytes, stream, (hipEvent_t)start_event, (hipEvent_t)stop_event);
}

int foremoe_ffn_down_fwd(const void* h, foremoe_dtype dtype, int32_t d, int32_t F, int32_t S,
                         const int32_t* slot_offset, const int32_t* slot_widx, int32_t W, const void* w_down,
                         int64_t n_cap, void* y_perm, void* workspace, size_t ws_bytes, void* stream) {
  return ffn_down_fwd_impl(h, dtype, d, F, S, slot_offset, slot_widx, W, w_down, n_cap, y_perm, workspace, ws_bytes,
                           stream, nullptr, nullptr);
}

int foremoe_ffn_down_fwd_timed(const void* h, foremoe_dtype dtype, int32_t d, int32_t F, int32_t S,
                               const int32_t* slot_offset, const int32_t* slot_widx, int32_t W, const void* w_down,
                               int64_t n_cap, void* y_perm, void* workspace, size_t ws_bytes, void* stream,
                               void* start_event, void* stop_event) {
  return ffn_down_fwd_impl(h, dtype, d, F, S, slot_offset, slot_widx, W, w_down, n_cap, y_perm, workspace, ws_bytes,
                           stream, (hipEvent_t)start_event, (hipEvent_t)stop_event);
}

int foremoe_ffn_down_dgrad(const void* dy_perm, const void* save_au, foremoe_dtype dtype, int32_t d, int32_t F,
                           int32_t S, const int32_t* slot_offset, const int32_t* slot_widx, int32_t W,
                           const void* w_down, int64_t n_cap, void* d_au, void* workspace, size_t ws_bytes,
                           void* stream) {
  return ffn_down_dgrad_impl(dy_perm, save_au, dtype, d, F, S, slot_offset, slot_widx, W, w_down, n_cap, d_au,
                             workspace, ws_bytes, stream, nullptr, nullptr);
}

int foremoe_ffn_down_dgrad_timed(const void* dy_perm, const void* save_au, foremoe_dtype dtype, int32_t d, int32_t F,
                                 int32_t S, const int32_t* slot_offset, const int32_t* slot_widx, int32_t W,
                                 const void* w_down, int64_t n_cap, void* d_au, void* workspace, size_t ws_bytes,
                                 void* stream, void* start_event, void* stop_event) {
  return ffn_down_dgrad_impl(dy_perm, save_au, dtype, d, F, S, slot_offset, slot_widx, W, w_down, n_cap, d_au,
                             workspace, ws_bytes, stream, (hipEvent_t)start_event, (hipEvent_t)stop_event);
}

int foremoe_ffn_gate_up_dgrad(const void* d_au, foremoe_dtype dtype, int32_t d, int32_t F, int32_t S,
                              const int32_t* slot_offset, const int32_t* slot_widx, int32_t W, const void* w_gate_up,
                              int64_t n_cap, void* dx_perm, void* workspace, size_t ws_bytes, void* stream) {
  return ffn_gate_up_dgrad_impl(d_au, dtype, d, F, S, slot_offset, slot_widx, W, w_gate_up, n_cap, dx_perm,
                                workspace, ws_bytes, stream, nullptr, nullptr);
}

int foremoe_ffn_gate_up_dgrad_timed(const void* d_au, foremoe_dtype dtype, int32_t d, int32_t F, int32_t S,
                                    const int32_t* slot_offset, const int32_t* slot_widx, int32_t W,
                                    const void* w_gate_up, int64_t n_cap, void* dx_perm, void* workspace,
                                    size_t ws_bytes, void* stream, void* start_event, void* stop_event) {
  return ffn_gate_up_dgrad_impl(d_au, dtype, d, F, S, slot_offset, slot_widx, W, w_gate_up, n_cap, dx_perm,
                                workspace, ws_bytes, stream, (hipEvent_t)start_event, (hipEvent_t)stop_event);
}

int foremoe_grouped_ffn_dgrad(const void* dy_perm, const void* save_au, foremoe_dtype dtype, int32_t d, int32_t F,
                              int32_t S, const int32_t* slot_offset, const int32_t* slot_widx, int32_t W,
                              const void* w_gate_up, const void* w_down, int64_t n_cap, void* d_au, void* dx_perm,
                              void* workspace, size_t ws_bytes, void* stream) {
  int rc = foremoe_ffn_down_dgrad(dy_perm, save_au, dtype, d, F, S, slot_offset, slot_widx, W, w_down, n_cap, d_au,
                                  workspace, ws_bytes, stream);
  if (rc) return rc;
  return foremoe_ffn_gate_up_dgrad(d_au, dtype, d, F, S, slot_offset, slot_widx, W, w_gate_up, n_cap, dx_perm,
                                   workspace, ws_bytes, stream);
}

// One weight-gradient GEMM over n steps' rows (every step: A [n_cap, M],
// B [n_cap, N], slot table), accumulated into dw [G, M, N].
static int wgrad_common(const char* who, const foremoe_wgrad_step* steps, int32_t n, int lda, int ldb, int M, int N,
                        foremoe_dtype dtype, int32_t G, int32_t part, int32_t parts, float* dw, void* ws,
                        size_t ws_bytes, void* stream) {
  REQUIRE(G >= 1 && G <= FOREMOE_MAX_SLOTS, "%s: G=%d out of range", who, G);
  REQUIRE(parts >= 1 && parts <= FOREMOE_MAX_WGRAD_STEPS && part >= 0 && part < parts,
          "%s: part %d of %d out of range", who, part, parts);
  REQUIRE(ws || ws_bytes == 0, "%s: ws is NULL but ws_bytes > 0", who);
  REQUIRE(n >= 0 && n <= FOREMOE_MAX_WGRAD_STEPS, "%s: n_steps=%d out of range", who, n);
  REQUIRE(n == 0 || steps, "%s: steps is NULL", who);
  int V = 0;
  bool any = false;
  for (int m = 0; m < n; ++m) {
    const foremoe_wgrad_step& t = steps[m];
    REQUIRE(t.S >= 0 && t.S <= FOREMOE_MAX_SLOTS, "%s: step %d: S=%d out of range", who, m, t.S);
    REQUIRE(t.n_cap >= 0 && t.n_cap < (int64_t)INT_MAX, "%s: step %d: n_cap out of range", who, m);
    if (t.S == 0 || t.n_cap == 0) continue;
    REQUIRE(t.a && t.b && t.slot_offset && t.slot_gidx, "%s: step %d: NULL buffer", who, m);
    if (dtype == FOREMOE_BF16 && (t.n_cap + 256) * (int64_t)(M > N ? M : N) * 2 >= ((int64_t)1 << 32))
      return set_error(FOREMOE_EUNSUPPORTED, "%s: step %d: (n_cap + 256) * row bytes must stay below 4 GiB", who, m);
    V += t.S;
    any = true;
  }
  REQUIRE(V <= FOREMOE_MAX_SLOTS, "%s: %d slots over all steps, at most %d", who, V, FOREMOE_MAX_SLOTS);
  if (!any) return FOREMOE_OK;
  REQUIRE(dw, "%s: NULL buffer", who);
  hipStream_t st = (hipStream_t)stream;
  if (dtype == FOREMOE_BF16) {
    WgradArgs a{};
    int v = 0;
    for (int m = 0; m < n; ++m) {
      const foremoe_wgrad_step& t = steps[m];
      if (t.S == 0 || t.n_cap == 0) continue;  // contributes nothing
      WgradStep& q = a.step[a.n_steps++];
      q.A = (const uint16_t*)t.a;
      q.B = (const uint16_t*)t.b;
      q.slot_offset = t.slot_offset;
      q.slot_gidx = t.slot_gidx;
      q.S = t.S;
      q.vbase = v;
      q.n_cap = t.n_cap;
      v += t.S;
    }
    a.V = v;
    a.tpart = part;
    a.tparts = parts;
    a.lda = lda;
    a.ldb = ldb;
    a.M = M;
    a.N = N;
    a.G = G;
    a.C = dw;
    a.ldc = N;
    a.gstride = (int64_t)M * N;
    // the workspace header holds the work counters; the rest partial tiles
    const bool has_ws = ws && ws_bytes >= kWgradHeaderBytes;
    const bool has_part = has_ws && ws_bytes >= kWgradHeaderBytes + kWgradPlanBytes;
    a.sched = has_ws ? (unsigned*)ws : nullptr;
    a.plan_out = has_part ? (int*)((char*)ws + kWgradHeaderBytes) : nullptr;
    a.part = has_part ? (float*)((char*)ws + kWgradHeaderBytes + kWgradPlanBytes) : nullptr;
    const size_t part_bytes = has_part ? ws_bytes - kWgradHeaderBytes - kWgradPlanBytes : 0;
    const dim3 grid(persistent_grid()), block(256);
    if (M % 256 == 0 && N % 256 == 0) {
      constexpr int WGM = FM_WG_WGM, WGN = FM_WG_WGN;
      a.p_max = (int)(part_bytes / (256 * 256 * 4));
      hipLaunchKernelGGL((gemm_wgrad_kernel<256, 256, FM_WG_BK, FM_WG_NS, WGM, WGN>), grid, dim3(64 * WGM * WGN), 0,
                         st, a);
      if (a.p_max > 0) hipLaunchKernelGGL((wgrad_reduce_kernel<256, 256, FM_WG_BK>), dim3(persistent_grid() * 4), block, 0, st, a);
    } else {
      a.p_max = (int)(part_bytes / (128 * 128 * 4));
      hipLaunchKernelGGL((gemm_wgrad_kernel<128, 128, 64, 3, 2, 2>), grid, block, 0, st, a);
      if (a.p_max > 0) hipLaunchKernelGGL((wgrad_reduce_kernel<128, 128, 64>), dim3(persistent_grid() * 4), block, 0, st, a);
    }
  } else {
    // fp32 path: one launch per step, in step order (each adds into dw);
    // a part is the rows m of dw with m % parts == part
    for (int m = 0; m < n; ++m) {
      const foremoe_wgrad_step& t = steps[m];
      if (t.S == 0 || t.n_cap == 0) continue;
      hipLaunchKernelGGL(f32_wgrad_kernel, dim3((N + 15) / 16, (M + 15) / 16, G), dim3(256), 0, st,
                         (const float*)t.a, lda, (const float*)t.b, ldb, M, N, t.slot_offset, t.slot_gidx, t.S, G,
                         t.n_cap, part, parts, dw);
    }
  }
  return check_launch(who);
}

static int check_wgrad_shape(const char* who, foremoe_dtype dtype, int32_t d, int32_t F) {
  REQUIRE(dtype == FOREMOE_F32 || dtype == FOREMOE_BF16, "%s: bad dtype", who);
  REQUIRE(d >= 1 && F >= 1, "%s: d and F must be positive", who);
  if (dtype == FOREMOE_BF16 && (d % 128 != 0 || F % 128 != 0))
    return set_error(FOREMOE_EUNSUPPORTED, "%s: bf16 needs d %% 128 == 0 and F %% 128 == 0 (d=%d, F=%d)", who, d, F);
  return FOREMOE_OK;
}

size_t foremoe_ffn_workspace_size(void) { return rows_workspace_bytes(); }

size_t foremoe_wgrad_workspace_size(int32_t d, int32_t F) {
  if (d < 1 || F < 1) return 0;
  return kWgradWorkspaceBytes;
}

int foremoe_ffn_gate_up_wgrad_steps(const foremoe_wgrad_step* steps, int32_t n_steps, foremoe_dtype dtype,
                                    int32_t d, int32_t F, int32_t G, int32_t part, int32_t parts, float* dw_gate_up,
                                    void* ws, size_t ws_bytes, void* stream) {
  int rc = check_wgrad_shape("gate_up_wgrad", dtype, d, F);
  if (rc) return rc;
  return wgrad_common("foremoe_ffn_gate_up_wgrad", steps, n_steps, 2 * F, d, 2 * F, d, dtype, G, part, parts,
                      dw_gate_up, ws, ws_bytes, stream);
}

int foremoe_ffn_down_wgrad_steps(const foremoe_wgrad_step* steps, int32_t n_steps, foremoe_dtype dtype, int32_t d,
                                 int32_t F, int32_t G, int32_t part, int32_t parts, float* dw_down, void* ws,
                                 size_t ws_bytes, void* stream) {
  int rc = check_wgrad_shape("down_wgrad", dtype, d, F);
  if (rc) return rc;
  return wgrad_common("foremoe_ffn_down_wgrad", steps, n_steps, d, F, d, F, dtype, G, part, parts, dw_down, ws,
                      ws_bytes, stream);
}

int foremoe_ffn_gate_up_wgrad(const void* d_au, const void* x_perm, foremoe_dtype dtype, int32_t d, int32_t F,
                              int32_t S, const int32_t* slot_offset, const int32_t* slot_gidx, int32_t G,
                              int64_t n_cap, float* dw_gate_up, void* ws, size_t ws_bytes, void* stream) {
  int rc = check_ffn("gate_up_wgrad", dtype, d, F, S, n_cap, slot_offset);
  if (rc) return rc;
  const foremoe_wgrad_step one = {d_au, x_perm, slot_offset, slot_gidx, S, n_cap};
  return foremoe_ffn_gate_up_wgrad_steps(&one, 1, dtype, d, F, G, 0, 1, dw_gate_up, ws, ws_bytes, stream);
}

int foremoe_ffn_down_wgrad(const void* dy_perm, const void* h, foremoe_dtype dtype, int32_t d, int32_t F, int32_t S,
                           const int32_t* slot_offset, const int32_t* slot_gidx, int32_t G, int64_t n_cap,
                           float* dw_down, void* ws, size_t ws_bytes, void* stream) {
  int rc = check_ffn("down_wgrad", dtype, d, F, S, n_cap, slot_offset);
  if (rc) return rc;
  const foremoe_wgrad_step one = {dy_perm, h, slot_offset, slot_gidx, S, n_cap};
  return foremoe_ffn_down_wgrad_steps(&one, 1, dtype, d, F, G, 0, 1, dw_down, ws, ws_bytes, stream);
}

int foremoe_grouped_ffn_wgrad(const void* x_perm, const void* h, const void* dy_perm, const void* d_au,
                              foremoe_dtype dtype, int32_t d, int32_t F, int32_t S, const int32_t* slot_offset,
                              const int32_t* slot_gidx, int32_t G, int64_t n_cap, float* dw_gate_up, float* dw_down,
                              void* ws, size_t ws_bytes, void* stream) {
  int rc = foremoe_ffn_gate_up_wgrad(d_au, x_perm, dtype, d, F, S, slot_offset, slot_gidx, G, n_cap, dw_gate_up, ws,
                                     ws_bytes, stream);
  if (rc) return rc;
  return foremoe_ffn_down_wgrad(dy_perm, h, dtype, d, F, S, slot_offset, slot_gidx, G, n_cap, dw_down, ws, ws_bytes,
                                stream);
}

}  // extern "C"
