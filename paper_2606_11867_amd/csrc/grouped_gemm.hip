// Step 4: grouped SwiGLU expert FFN over the local slots (App. A), forward,
// input gradient and weight gradient.
//
// bf16 path: persistent workgroups of 4 wavefronts walk a tile list built on
// the device from the slot offsets (no host sync), stage 64-deep K slices of
// both operands through double-buffered LDS, and multiply with
// v_mfma_f32_32x32x16_bf16 (fp32 accumulation). The SwiGLU activation and
// its derivative are fused into the epilogues. Operands that are contiguous
// along M/N (the weight-gradient operands and the transposed weights of the
// input gradient) are transposed 8x8 in registers on their way to LDS, so
// LDS always holds K-contiguous rows for the MFMA reads.
//
// f32 path: plain per-element kernels (small shapes only; no MFMA).
#include <climits>

#include "common.h"

namespace foremoe {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kThreads = 256;
constexpr int kBK = 64;
constexpr int kStr = kBK + 8;  // LDS row stride in elements (144 bytes: conflict-free MFMA reads)

enum Epi { kEpiStore = 0, kEpiSwigluFwd = 1, kEpiSwigluBwd = 2, kEpiAccF32 = 3 };

__device__ __forceinline__ float silu_f(float a) { return a / (1.0f + __expf(-a)); }

// Virtual workgroup id: workgroups are dispatched round-robin over the 8 XCDs,
// so give the workgroups of one XCD consecutive ids (they then share tiles
// that reuse the same operand rows in that XCD's L2).
__device__ __forceinline__ int xcd_virtual_id() {
  const int b = blockIdx.x, n = gridDim.x;
  if (n % 8 != 0) return b;
  return (b % 8) * (n / 8) + b / 8;
}

// Block-wide inclusive scan (256 threads).
__device__ int scan256(int v, int* s_tmp, int& total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int n = __shfl_up(v, o, 64);
    if (lane >= o) v += n;
  }
  if (lane == 63) s_tmp[w] = v;
  __syncthreads();
  int before = 0;
  total = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int t = s_tmp[i];
    if (i < w) before += t;
    total += t;
  }
  __syncthreads();
  return v + before;
}

// ---------------------------------------------------------------------------
// Tile loaders (global -> registers -> LDS)
// ---------------------------------------------------------------------------
// ROWS x 64 tile whose rows are K-contiguous in global memory. Thread t moves
// 16 bytes of row (t / 8 + 32 p), column (t % 8) * 8, for p < ROWS / 32.
template <int ROWS>
struct KcLoader {
  static constexpr int NP = ROWS / 32;
  const uint16_t* ptr[NP];
  uint4 v[NP];
  __device__ __forceinline__ int row(int p) const { return p * 32 + (threadIdx.x >> 3); }
  __device__ __forceinline__ int col() const { return (threadIdx.x & 7) * 8; }
  __device__ __forceinline__ void load(int k0) {
#pragma unroll
    for (int p = 0; p < NP; ++p) v[p] = *reinterpret_cast<const uint4*>(ptr[p] + k0 + col());
  }
  __device__ __forceinline__ void store(uint16_t* s) const {
#pragma unroll
    for (int p = 0; p < NP; ++p) *reinterpret_cast<uint4*>(s + row(p) * kStr + col()) = v[p];
  }
};

// ROWS x 64 tile stored K-major in global memory: element (r, k) at
// base + k * ld + r. Each thread loads 8x8 blocks (8 K rows of 8 contiguous
// elements), transposes them in registers and writes 8 K-contiguous LDS rows.
// K rows outside [lo, hi) read as zero.
template <int ROWS>
struct McLoader {
  static constexpr int KB = kBK / 8;
  static constexpr int NBLK = KB * (ROWS / 8);
  static constexpr int PER = (NBLK + kThreads - 1) / kThreads;
  uint4 v[PER][8];
  __device__ __forceinline__ int blk(int b) const { return b * kThreads + threadIdx.x; }
  __device__ __forceinline__ void load(const uint16_t* base, int64_t ld, int k0, int lo, int hi) {
#pragma unroll
    for (int b = 0; b < PER; ++b) {
      const int id = blk(b);
      if (NBLK % kThreads != 0 && id >= NBLK) continue;
      const int kb = id % KB, mb = id / KB;
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        const int k = k0 + kb * 8 + r;
        if (k >= lo && k < hi)
          v[b][r] = *reinterpret_cast<const uint4*>(base + (int64_t)k * ld + mb * 8);
        else
          v[b][r] = make_uint4(0, 0, 0, 0);
      }
    }
  }
  __device__ __forceinline__ void store(uint16_t* s) const {
#pragma unroll
    for (int b = 0; b < PER; ++b) {
      const int id = blk(b);
      if (NBLK % kThreads != 0 && id >= NBLK) continue;
      const int kb = id % KB, mb = id / KB;
      uint32_t w[8][4];
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        w[r][0] = v[b][r].x;
        w[r][1] = v[b][r].y;
        w[r][2] = v[b][r].z;
        w[r][3] = v[b][r].w;
      }
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        const uint32_t sel = (c & 1) ? 0x07060302u : 0x05040100u;
        uint32_t o[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) o[i] = __builtin_amdgcn_perm(w[2 * i + 1][c >> 1], w[2 * i][c >> 1], sel);
        *reinterpret_cast<uint4*>(s + (mb * 8 + c) * kStr + kb * 8) = make_uint4(o[0], o[1], o[2], o[3]);
      }
    }
  }
};

// ---------------------------------------------------------------------------
// MFMA tile core: 4 wavefronts as 2 x 2, each owning (BM/2) x (BN/2) of the
// output as 32x32 blocks. The MFMA is fed the B rows as its first operand,
// so each lane ends up with 4 consecutive output columns of one output row:
// block (i, j), register q of lane l holds row  wm*BM/2 + 32 i + l % 32  and
// column  col(j) + 8 (q / 4) + 4 (l / 32) + q % 4.
// ---------------------------------------------------------------------------
template <int BM, int BN, bool SWIGLU_COLS>
struct Core {
  static constexpr int WM = BM / 2, WN = BN / 2;
  static constexpr int MB = WM / 32, NB = WN / 32;
  f32x16 acc[MB][NB];

  // LDS row of the B tile that wave column wn's block j starts at.
  __device__ __forceinline__ static int bcol(int wn, int j) {
    if constexpr (SWIGLU_COLS) {
      // gate rows live in [0, BN/2), up rows in [BN/2, BN); the wave keeps the
      // gate block j and the up block j + NB/2 of the same output columns
      constexpr int H = NB / 2;
      return j < H ? wn * (BN / 4) + j * 32 : BN / 2 + wn * (BN / 4) + (j - H) * 32;
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

  __device__ __forceinline__ void compute(const uint16_t* As, const uint16_t* Bs, int wm, int wn) {
    const int lane = threadIdx.x & 63;
    const int l32 = lane & 31, hi8 = (lane >> 5) * 8;
#pragma unroll
    for (int kk = 0; kk < kBK / 16; ++kk) {
      bf16x8 af[MB], bfr[NB];
#pragma unroll
      for (int i = 0; i < MB; ++i)
        af[i] = *reinterpret_cast<const bf16x8*>(As + (wm * WM + i * 32 + l32) * kStr + kk * 16 + hi8);
#pragma unroll
      for (int j = 0; j < NB; ++j)
        bfr[j] = *reinterpret_cast<const bf16x8*>(Bs + (bcol(wn, j) + l32) * kStr + kk * 16 + hi8);
#pragma unroll
      for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int j = 0; j < NB; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[j], af[i], acc[i][j], 0, 0, 0);
    }
  }
};

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
};

// Per-slot m-tile prefix in LDS: s_mt[j] = m-tiles of slots before j.
template <int BM>
__device__ void build_slot_tiles(const int32_t* __restrict__ off, int S, int64_t n_cap, int* s_mt, int* s_tmp) {
  int carry = 0;
  for (int j0 = 0; j0 < S; j0 += kThreads) {
    const int j = j0 + threadIdx.x;
    int n = 0;
    if (j < S) {
      int64_t lo = off[j], hi = off[j + 1];
      lo = lo < 0 ? 0 : (lo > n_cap ? n_cap : lo);
      hi = hi < 0 ? 0 : (hi > n_cap ? n_cap : hi);
      n = hi > lo ? (int)((hi - lo + BM - 1) / BM) : 0;
    }
    int total;
    const int incl = scan256(n, s_tmp, total);
    if (j < S) s_mt[j] = carry + incl - n;
    carry += total;
  }
  if (threadIdx.x == 0) s_mt[S] = carry;
  __syncthreads();
}

template <int BM, int BN, bool B_KCONTIG, int EPI>
__global__ __launch_bounds__(kThreads) void gemm_rows_kernel(RowsArgs a) {
  constexpr bool SW = (EPI == kEpiSwigluFwd);
  __shared__ __attribute__((aligned(16))) uint16_t lds[2][(BM + BN) * kStr];
  __shared__ int s_mt[FOREMOE_MAX_SLOTS + 1];
  __shared__ int s_tmp[4];

  build_slot_tiles<BM>(a.slot_offset, a.S, a.n_cap, s_mt, s_tmp);
  const int n_tiles = a.N / BN;
  const int total = s_mt[a.S] * n_tiles;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int KT = a.K / kBK;

  Core<BM, BN, SW> core;
  KcLoader<BM> la;
  KcLoader<BN> lbk;
  McLoader<BN> lbm;

  for (int t = xcd_virtual_id(); t < total; t += gridDim.x) {
    const int mtg = t / n_tiles, nt = t % n_tiles;
    int lo = 0, hi = a.S - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (s_mt[mid] <= mtg) lo = mid;
      else hi = mid - 1;
    }
    const int j = lo;
    int64_t rbeg = a.slot_offset[j], rend = a.slot_offset[j + 1];
    rbeg = rbeg < 0 ? 0 : (rbeg > a.n_cap ? a.n_cap : rbeg);
    rend = rend < 0 ? 0 : (rend > a.n_cap ? a.n_cap : rend);
    const int64_t m0 = rbeg + (int64_t)(mtg - s_mt[j]) * BM;
    const int w = a.slot_widx[j];
    if (w < 0 || w >= a.W) continue;  // invalid weight index: rows left unwritten
    const uint16_t* Bw = a.B + (int64_t)w * a.wstride;
    const int n0 = nt * BN;           // first output column of the tile grid
    const int f0 = nt * (BN / 2);     // SwiGLU: first H column

#pragma unroll
    for (int p = 0; p < KcLoader<BM>::NP; ++p) {
      int64_t r = m0 + la.row(p);
      if (r >= rend) r = rend - 1;  // clamp the ragged tail to a valid row
      la.ptr[p] = a.A + r * a.lda;
    }
    if constexpr (B_KCONTIG) {
#pragma unroll
      for (int p = 0; p < KcLoader<BN>::NP; ++p) {
        const int r = lbk.row(p);
        int64_t wr;
        if constexpr (SW) wr = r < BN / 2 ? f0 + r : a.F + f0 + (r - BN / 2);
        else wr = n0 + r;
        lbk.ptr[p] = Bw + wr * a.ldb;
      }
    }
    const uint16_t* Bkn = Bw + n0;  // K-major weights: element (n, k) at Bkn + k * ldb + n

    core.zero();
    la.load(0);
    if constexpr (B_KCONTIG) lbk.load(0);
    else lbm.load(Bkn, a.ldb, 0, 0, a.K);
    la.store(lds[0]);
    if constexpr (B_KCONTIG) lbk.store(lds[0] + BM * kStr);
    else lbm.store(lds[0] + BM * kStr);
    __syncthreads();
    for (int kt = 0; kt < KT; ++kt) {
      const int cur = kt & 1;
      const bool more = kt + 1 < KT;
      if (more) {
        la.load((kt + 1) * kBK);
        if constexpr (B_KCONTIG) lbk.load((kt + 1) * kBK);
        else lbm.load(Bkn, a.ldb, (kt + 1) * kBK, 0, a.K);
      }
      core.compute(lds[cur], lds[cur] + BM * kStr, wm, wn);
      if (more) {
        la.store(lds[cur ^ 1]);
        if constexpr (B_KCONTIG) lbk.store(lds[cur ^ 1] + BM * kStr);
        else lbm.store(lds[cur ^ 1] + BM * kStr);
      }
      __syncthreads();
    }

    // ---------------- epilogue ----------------
    const int l32 = lane & 31, c4 = (lane >> 5) * 4;
#pragma unroll
    for (int i = 0; i < Core<BM, BN, SW>::MB; ++i) {
      const int64_t row = m0 + wm * (BM / 2) + i * 32 + l32;
      if (row >= rend) continue;
      if constexpr (EPI == kEpiSwigluFwd) {
        constexpr int H = Core<BM, BN, SW>::NB / 2;
#pragma unroll
        for (int jj = 0; jj < H; ++jj) {
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const int f = f0 + wn * (BN / 4) + jj * 32 + g * 8 + c4;
            float hv[4], av[4], uv[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              av[e] = core.acc[i][jj][g * 4 + e];
              uv[e] = core.acc[i][jj + H][g * 4 + e];
              hv[e] = silu_f(av[e]) * uv[e];
            }
            *reinterpret_cast<uint2*>(a.C + row * a.ldc + f) = make_uint2(pack_bf2(hv[0], hv[1]), pack_bf2(hv[2], hv[3]));
            if (a.C2) {
              *reinterpret_cast<uint2*>(a.C2 + row * a.ldc2 + f) =
                  make_uint2(pack_bf2(av[0], av[1]), pack_bf2(av[2], av[3]));
              *reinterpret_cast<uint2*>(a.C2 + row * a.ldc2 + a.F + f) =
                  make_uint2(pack_bf2(uv[0], uv[1]), pack_bf2(uv[2], uv[3]));
            }
          }
        }
      } else {
#pragma unroll
        for (int jj = 0; jj < Core<BM, BN, SW>::NB; ++jj) {
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const int n = n0 + wn * (BN / 2) + jj * 32 + g * 8 + c4;
            float v[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = core.acc[i][jj][g * 4 + e];
            if constexpr (EPI == kEpiSwigluBwd) {
              // v = dH at columns f = n..n+3; saved A in [0, F), U in [F, 2F)
              const uint2 ra = *reinterpret_cast<const uint2*>(a.AU + row * a.ldau + n);
              const uint2 ru = *reinterpret_cast<const uint2*>(a.AU + row * a.ldau + a.F + n);
              const float A4[4] = {bf2f(ra.x & 0xFFFF), bf2f(ra.x >> 16), bf2f(ra.y & 0xFFFF), bf2f(ra.y >> 16)};
              const float U4[4] = {bf2f(ru.x & 0xFFFF), bf2f(ru.x >> 16), bf2f(ru.y & 0xFFFF), bf2f(ru.y >> 16)};
              float da[4], du[4];
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                const float s = 1.0f / (1.0f + __expf(-A4[e]));
                da[e] = v[e] * U4[e] * (s + A4[e] * s * (1.0f - s));
                du[e] = v[e] * A4[e] * s;
              }
              *reinterpret_cast<uint2*>(a.C + row * a.ldc + n) = make_uint2(pack_bf2(da[0], da[1]), pack_bf2(da[2], da[3]));
              *reinterpret_cast<uint2*>(a.C + row * a.ldc + a.F + n) =
                  make_uint2(pack_bf2(du[0], du[1]), pack_bf2(du[2], du[3]));
            } else {
              *reinterpret_cast<uint2*>(a.C + row * a.ldc + n) = make_uint2(pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3]));
            }
          }
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Weight gradient: dW[g] (M x N, fp32) += sum over the rows of every slot
// with gradient index g of A[row, :]^T B[row, :]. Groups are visited in
// descending row count so that the long reductions start first.
// ---------------------------------------------------------------------------
struct WgradArgs {
  const uint16_t* A;  // [n_cap, M]
  int64_t lda;
  const uint16_t* B;  // [n_cap, N]
  int64_t ldb;
  int M, N;
  const int32_t* slot_offset;
  const int32_t* slot_gidx;
  int S, G;
  int64_t n_cap;
  float* C;  // dW[g] at C + g * gstride, row-major [M, N]
  int64_t ldc;
  int64_t gstride;
};

template <int BM, int BN>
__global__ __launch_bounds__(kThreads) void gemm_wgrad_kernel(WgradArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t lds[2][(BM + BN) * kStr];
  __shared__ int s_off[FOREMOE_MAX_SLOTS + 1];
  __shared__ int s_gidx[FOREMOE_MAX_SLOTS];
  __shared__ int s_rows[FOREMOE_MAX_SLOTS];
  __shared__ int s_order[FOREMOE_MAX_SLOTS];
  __shared__ int s_nne;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int S = a.S, G = a.G;
  if (tid == 0) s_nne = 0;
  for (int g = tid; g < G; g += kThreads) s_rows[g] = 0;
  for (int j = tid; j <= S; j += kThreads) {
    int64_t o = a.slot_offset[j];
    s_off[j] = (int)(o < 0 ? 0 : (o > a.n_cap ? a.n_cap : o));
    if (j < S) {
      const int g = a.slot_gidx[j];
      s_gidx[j] = (g >= 0 && g < G) ? g : -1;
    }
  }
  __syncthreads();
  for (int j = tid; j < S; j += kThreads) {
    const int n = s_off[j + 1] - s_off[j];
    if (n <= 0) s_gidx[j] = -1;  // empty (or inverted) ranges contribute nothing
    else if (s_gidx[j] >= 0) atomicAdd(&s_rows[s_gidx[j]], n);
  }
  __syncthreads();
  for (int g = tid; g < G; g += kThreads) {
    const int rg = s_rows[g];
    if (rg <= 0) continue;
    int rank = 0;
    for (int h = 0; h < G; ++h) {
      const int rh = s_rows[h];
      rank += (rh > rg) || (rh == rg && h < g);
    }
    s_order[rank] = g;
    atomicAdd(&s_nne, 1);
  }
  __syncthreads();

  const int mt_n = a.M / BM, nt_n = a.N / BN, tpg = mt_n * nt_n;
  const int total = s_nne * tpg;
  Core<BM, BN, false> core;
  McLoader<BM> la;
  McLoader<BN> lb;

  for (int t = xcd_virtual_id(); t < total; t += gridDim.x) {
    const int g = s_order[t / tpg];
    const int tt = t % tpg;
    const int m0 = (tt / nt_n) * BM, n0 = (tt % nt_n) * BN;
    const uint16_t* Ab = a.A + m0;
    const uint16_t* Bb = a.B + n0;

    int j = 0;
    while (j < S && !(s_gidx[j] == g && s_off[j + 1] > s_off[j])) ++j;
    int k0 = s_off[j];

    core.zero();
    la.load(Ab, a.lda, k0, s_off[j], s_off[j + 1]);
    lb.load(Bb, a.ldb, k0, s_off[j], s_off[j + 1]);
    la.store(lds[0]);
    lb.store(lds[0] + BM * kStr);
    __syncthreads();
    int cur = 0;
    while (true) {
      int j2 = j, k2 = k0 + kBK;
      if (k2 >= s_off[j + 1]) {
        ++j2;
        while (j2 < S && !(s_gidx[j2] == g && s_off[j2 + 1] > s_off[j2])) ++j2;
        k2 = j2 < S ? s_off[j2] : 0;
      }
      const bool more = j2 < S;
      if (more) {
        la.load(Ab, a.lda, k2, s_off[j2], s_off[j2 + 1]);
        lb.load(Bb, a.ldb, k2, s_off[j2], s_off[j2 + 1]);
      }
      core.compute(lds[cur], lds[cur] + BM * kStr, wm, wn);
      if (more) {
        la.store(lds[cur ^ 1]);
        lb.store(lds[cur ^ 1] + BM * kStr);
      }
      __syncthreads();
      if (!more) break;
      cur ^= 1;
      j = j2;
      k0 = k2;
    }

    float* Cg = a.C + (int64_t)g * a.gstride;
    const int l32 = lane & 31, c4 = (lane >> 5) * 4;
#pragma unroll
    for (int i = 0; i < Core<BM, BN, false>::MB; ++i) {
      const int64_t m = m0 + wm * (BM / 2) + i * 32 + l32;
#pragma unroll
      for (int jj = 0; jj < Core<BM, BN, false>::NB; ++jj) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int n = n0 + wn * (BN / 2) + jj * 32 + q * 8 + c4;
          float4* p = reinterpret_cast<float4*>(Cg + m * a.ldc + n);
          float4 o = *p;
          o.x += core.acc[i][jj][q * 4 + 0];
          o.y += core.acc[i][jj][q * 4 + 1];
          o.z += core.acc[i][jj][q * 4 + 2];
          o.w += core.acc[i][jj][q * 4 + 3];
          *p = o;
        }
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
                                                        float* __restrict__ C) {
  const int n = blockIdx.x * 16 + (threadIdx.x & 15);
  const int m = blockIdx.y * 16 + (threadIdx.x >> 4);
  const int g = blockIdx.z;
  if (n >= N || m >= M) return;
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

template <int BN, bool KC, int EPI>
void launch_rows(const RowsArgs& a, hipStream_t st) {
  hipLaunchKernelGGL((gemm_rows_kernel<256, BN, KC, EPI>), dim3(persistent_grid()), dim3(kThreads), 0, st, a);
}

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
  return FOREMOE_OK;
}

static dim3 f32_grid(int cols, int64_t rows) {
  return dim3((unsigned)((cols + 15) / 16), (unsigned)((rows + 15) / 16 > 0 ? (rows + 15) / 16 : 1));
}

extern "C" {

int foremoe_ffn_gate_up_fwd(const void* x_perm, foremoe_dtype dtype, int32_t d, int32_t F, int32_t S,
                            const int32_t* slot_offset, const int32_t* slot_widx, int32_t W, const void* w_gate_up,
                            int64_t n_cap, void* h, void* save_au, void* stream) {
  int rc = check_ffn("gate_up_fwd", dtype, d, F, S, n_cap, slot_offset);
  if (rc) return rc;
  if (S == 0 || n_cap == 0) return FOREMOE_OK;
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
    launch_rows<256, true, kEpiSwigluFwd>(a, st);
  } else {
    hipLaunchKernelGGL(f32_rows_kernel<kF32GateUpFwd>, f32_grid(F, n_cap), dim3(256), 0, st, (const float*)x_perm,
                       (const float*)w_gate_up, nullptr, d, F, W, slot_offset, slot_widx, S, n_cap, (float*)h,
                       (float*)save_au);
  }
  return check_launch("foremoe_ffn_gate_up_fwd");
}

int foremoe_ffn_down_fwd(const void* h, foremoe_dtype dtype, int32_t d, int32_t F, int32_t S,
                         const int32_t* slot_offset, const int32_t* slot_widx, int32_t W, const void* w_down,
                         int64_t n_cap, void* y_perm, void* stream) {
  int rc = check_ffn("down_fwd", dtype, d, F, S, n_cap, slot_offset);
  if (rc) return rc;
  if (S == 0 || n_cap == 0) return FOREMOE_OK;
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
    if (d % 256 == 0) launch_rows<256, true, kEpiStore>(a, st);
    else launch_rows<128, true, kEpiStore>(a, st);
  } else {
    hipLaunchKernelGGL(f32_rows_kernel<kF32DownFwd>, f32_grid(d, n_cap), dim3(256), 0, st, (const float*)h,
                       (const float*)w_down, nullptr, d, F, W, slot_offset, slot_widx, S, n_cap, (float*)y_perm,
                       nullptr);
  }
  return check_launch("foremoe_ffn_down_fwd");
}

int foremoe_grouped_ffn_fwd(const void* x_perm, foremoe_dtype dtype, int32_t d, int32_t F, int32_t S,
                            const int32_t* slot_offset, const int32_t* slot_widx, int32_t W, const void* w_gate_up,
                            const void* w_down, int64_t n_cap, void* h, void* y_perm, void* save_au, void* stream) {
  int rc = foremoe_ffn_gate_up_fwd(x_perm, dtype, d, F, S, slot_offset, slot_widx, W, w_gate_up, n_cap, h, save_au,
                                   stream);
  if (rc) return rc;
  return foremoe_ffn_down_fwd(h, dtype, d, F, S, slot_offset, slot_widx, W, w_down, n_cap, y_perm, stream);
}

int foremoe_ffn_down_dgrad(const void* dy_perm, const void* save_au, foremoe_dtype dtype, int32_t d, int32_t F,
                           int32_t S, const int32_t* slot_offset, const int32_t* slot_widx, int32_t W,
                           const void* w_down, int64_t n_cap, void* d_au, void* stream) {
  int rc = check_ffn("down_dgrad", dtype, d, F, S, n_cap, slot_offset);
  if (rc) return rc;
  if (S == 0 || n_cap == 0) return FOREMOE_OK;
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
    if (F % 256 == 0) launch_rows<256, false, kEpiSwigluBwd>(a, st);
    else launch_rows<128, false, kEpiSwigluBwd>(a, st);
  } else {
    hipLaunchKernelGGL(f32_rows_kernel<kF32DownDgrad>, f32_grid(F, n_cap), dim3(256), 0, st, (const float*)dy_perm,
                       (const float*)w_down, (const float*)save_au, d, F, W, slot_offset, slot_widx, S, n_cap,
                       (float*)d_au, nullptr);
  }
  return check_launch("foremoe_ffn_down_dgrad");
}

int foremoe_ffn_gate_up_dgrad(const void* d_au, foremoe_dtype dtype, int32_t d, int32_t F, int32_t S,
                              const int32_t* slot_offset, const int32_t* slot_widx, int32_t W, const void* w_gate_up,
                              int64_t n_cap, void* dx_perm, void* stream) {
  int rc = check_ffn("gate_up_dgrad", dtype, d, F, S, n_cap, slot_offset);
  if (rc) return rc;
  if (S == 0 || n_cap == 0) return FOREMOE_OK;
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
    if (d % 256 == 0) launch_rows<256, false, kEpiStore>(a, st);
    else launch_rows<128, false, kEpiStore>(a, st);
  } else {
    hipLaunchKernelGGL(f32_rows_kernel<kF32GateUpDgrad>, f32_grid(d, n_cap), dim3(256), 0, st, (const float*)d_au,
                       (const float*)w_gate_up, nullptr, d, F, W, slot_offset, slot_widx, S, n_cap, (float*)dx_perm,
                       nullptr);
  }
  return check_launch("foremoe_ffn_gate_up_dgrad");
}

int foremoe_grouped_ffn_dgrad(const void* dy_perm, const void* save_au, foremoe_dtype dtype, int32_t d, int32_t F,
                              int32_t S, const int32_t* slot_offset, const int32_t* slot_widx, int32_t W,
                              const void* w_gate_up, const void* w_down, int64_t n_cap, void* d_au, void* dx_perm,
                              void* stream) {
  int rc = foremoe_ffn_down_dgrad(dy_perm, save_au, dtype, d, F, S, slot_offset, slot_widx, W, w_down, n_cap, d_au,
                                  stream);
  if (rc) return rc;
  return foremoe_ffn_gate_up_dgrad(d_au, dtype, d, F, S, slot_offset, slot_widx, W, w_gate_up, n_cap, dx_perm,
                                   stream);
}

static int wgrad_common(const char* who, const void* A, int lda, const void* B, int ldb, int M, int N,
                        foremoe_dtype dtype, int32_t S, const int32_t* slot_offset, const int32_t* slot_gidx, int32_t G,
                        int64_t n_cap, float* dw, void* stream) {
  REQUIRE(G >= 1 && G <= FOREMOE_MAX_SLOTS, "%s: G=%d out of range", who, G);
  if (S == 0 || n_cap == 0) return FOREMOE_OK;
  REQUIRE(A && B && slot_gidx && dw, "%s: NULL buffer", who);
  hipStream_t st = (hipStream_t)stream;
  if (dtype == FOREMOE_BF16) {
    WgradArgs a{};
    a.A = (const uint16_t*)A;
    a.lda = lda;
    a.B = (const uint16_t*)B;
    a.ldb = ldb;
    a.M = M;
    a.N = N;
    a.slot_offset = slot_offset;
    a.slot_gidx = slot_gidx;
    a.S = S;
    a.G = G;
    a.n_cap = n_cap;
    a.C = dw;
    a.ldc = N;
    a.gstride = (int64_t)M * N;
    hipLaunchKernelGGL((gemm_wgrad_kernel<128, 128>), dim3(persistent_grid()), dim3(kThreads), 0, st, a);
  } else {
    hipLaunchKernelGGL(f32_wgrad_kernel, dim3((N + 15) / 16, (M + 15) / 16, G), dim3(256), 0, st, (const float*)A, lda,
                       (const float*)B, ldb, M, N, slot_offset, slot_gidx, S, G, n_cap, dw);
  }
  return check_launch(who);
}

int foremoe_ffn_gate_up_wgrad(const void* d_au, const void* x_perm, foremoe_dtype dtype, int32_t d, int32_t F,
                              int32_t S, const int32_t* slot_offset, const int32_t* slot_gidx, int32_t G,
                              int64_t n_cap, float* dw_gate_up, void* stream) {
  int rc = check_ffn("gate_up_wgrad", dtype, d, F, S, n_cap, slot_offset);
  if (rc) return rc;
  return wgrad_common("foremoe_ffn_gate_up_wgrad", d_au, 2 * F, x_perm, d, 2 * F, d, dtype, S, slot_offset, slot_gidx,
                      G, n_cap, dw_gate_up, stream);
}

int foremoe_ffn_down_wgrad(const void* dy_perm, const void* h, foremoe_dtype dtype, int32_t d, int32_t F, int32_t S,
                           const int32_t* slot_offset, const int32_t* slot_gidx, int32_t G, int64_t n_cap,
                           float* dw_down, void* stream) {
  int rc = check_ffn("down_wgrad", dtype, d, F, S, n_cap, slot_offset);
  if (rc) return rc;
  return wgrad_common("foremoe_ffn_down_wgrad", dy_perm, d, h, F, d, F, dtype, S, slot_offset, slot_gidx, G, n_cap,
                      dw_down, stream);
}

int foremoe_grouped_ffn_wgrad(const void* x_perm, const void* h, const void* dy_perm, const void* d_au,
                              foremoe_dtype dtype, int32_t d, int32_t F, int32_t S, const int32_t* slot_offset,
                              const int32_t* slot_gidx, int32_t G, int64_t n_cap, float* dw_gate_up, float* dw_down,
                              void* stream) {
  int rc = foremoe_ffn_gate_up_wgrad(d_au, x_perm, dtype, d, F, S, slot_offset, slot_gidx, G, n_cap, dw_gate_up,
                                     stream);
  if (rc) return rc;
  return foremoe_ffn_down_wgrad(dy_perm, h, dtype, d, F, S, slot_offset, slot_gidx, G, n_cap, dw_down, stream);
}

}  // extern "C"
