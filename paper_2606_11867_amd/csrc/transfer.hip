// The one-GPU half of the Expert Transfer Engine (Sec. 6): Copy-out and
// Copy-in of the policy-update swap (Sec. 6.2) and the CPU-assisted prefetch
// of experts from a pinned host master copy (Sec. 6.1).
//
// Copy-out packs the parameters and/or gradients of departing experts into
// one contiguous send buffer, one record per expert (App. A.3: S_e + S_g
// bytes): gate/up parameters [2F, d], down parameters [d, F], then the fp32
// gate/up and down gradients. Copy-in unpacks a receive buffer: parameters
// into their weight slots, gradients either moved into a slot (assign) or
// accumulated into the main expert's gradient (add; Sec. 6.2), records that
// name one gradient applied in record order in fp32, so the result is
// deterministic. Both kernels are HBM-bound copies moving 16-byte vectors
// with the nontemporal hint (the data streams through once); every record
// boundary and part boundary is a multiple of 16 bytes.
//
// The prefetch is a host-to-device DMA (hipMemcpyAsync on the caller's
// stream) straight into the weight slots: no kernel and no GPU buffer.
#include <algorithm>
#include <climits>
#include <vector>

#include "common.h"

namespace foremoe {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kXferThreads = 256;
constexpr int kXferVecPerThread = 4;  // 16-byte vectors per thread per pass, all loads before the stores

struct XferRecords {
  int32_t widx[FOREMOE_MAX_XFER_RECORDS];
  int32_t gidx[FOREMOE_MAX_XFER_RECORDS];
};

// Byte sizes of the four parts of a record; a part of size 0 is absent.
struct RecordParts {
  uint64_t gu_p, dn_p, gu_g, dn_g;  // gate/up params, down params, gate/up grads, down grads
  __host__ __device__ uint64_t total() const { return gu_p + dn_p + gu_g + dn_g; }
};

RecordParts record_parts(int d, int F, int p_w, int what) {
  RecordParts r{0, 0, 0, 0};
  if (what & FOREMOE_XFER_PARAMS) {
    r.gu_p = (uint64_t)2 * F * d * p_w;
    r.dn_p = (uint64_t)d * F * p_w;
  }
  if (what & FOREMOE_XFER_GRADS) {
    r.gu_g = (uint64_t)2 * F * d * 4;
    r.dn_g = (uint64_t)d * F * 4;
  }
  return r;
}

// Source (copy-out) or destination (copy-in) address of byte `off` of
// record r's memory in the expert arrays.
__device__ __forceinline__ char* part_addr(const RecordParts& rp, uint64_t off, int r, const XferRecords& rec,
                                           char* wgu, char* wdn, char* ggu, char* gdn) {
  if (off < rp.gu_p) return wgu + (uint64_t)rec.widx[r] * rp.gu_p + off;
  off -= rp.gu_p;
  if (off < rp.dn_p) return wdn + (uint64_t)rec.widx[r] * rp.dn_p + off;
  off -= rp.dn_p;
  if (off < rp.gu_g) return ggu + (uint64_t)rec.gidx[r] * rp.gu_g + off;
  off -= rp.gu_g;
  return gdn + (uint64_t)rec.gidx[r] * rp.dn_g + off;
}

// Copy-out: record r = blockIdx.y. Each thread moves kXferVecPerThread
// vectors per pass, issuing every load before the first store.
__global__ __launch_bounds__(kXferThreads) void copy_out_kernel(RecordParts rp, XferRecords rec, const char* wgu,
                                                                const char* wdn, const char* ggu, const char* gdn,
                                                                char* buf) {
  const int r = blockIdx.y;
  const uint64_t nvec = rp.total() / 16;
  char* dst = buf + (uint64_t)r * rp.total();
  const uint64_t step = (uint64_t)gridDim.x * kXferThreads * kXferVecPerThread;
  for (uint64_t v0 = (uint64_t)blockIdx.x * kXferThreads * kXferVecPerThread + threadIdx.x; v0 < nvec; v0 += step) {
    u32x4 a[kXferVecPerThread];
#pragma unroll
    for (int u = 0; u < kXferVecPerThread; ++u) {
      const uint64_t v = v0 + (uint64_t)u * kXferThreads;
      if (v < nvec)
        a[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(
            part_addr(rp, v * 16, r, rec, (char*)wgu, (char*)wdn, (char*)ggu, (char*)gdn)));
    }
#pragma unroll
    for (int u = 0; u < kXferVecPerThread; ++u) {
      const uint64_t v = v0 + (uint64_t)u * kXferThreads;
      if (v < nvec) __builtin_nontemporal_store(a[u], reinterpret_cast<u32x4*>(dst + v * 16));
    }
  }
}

// Copy-in work: rows [0, n_par) copy record par[i]'s parameters into weight
// slot widx of that record; rows [n_par, n_par + n_grp) each produce one
// gradient target: start from the record grp_start (assign) or from the
// target's current value (grp_start < 0), then add the records
// ord[grp_off[g]] .. ord[grp_off[g + 1] - 1] in that order, in fp32.
struct CopyInPlan {
  int32_t n_par, n_grp;
  int32_t par[FOREMOE_MAX_XFER_RECORDS];
  int32_t grp_tgt[FOREMOE_MAX_XFER_RECORDS];
  int32_t grp_start[FOREMOE_MAX_XFER_RECORDS];
  int32_t grp_off[FOREMOE_MAX_XFER_RECORDS + 1];
  int32_t ord[FOREMOE_MAX_XFER_RECORDS];
};

__device__ __forceinline__ float4 add4(float4 a, float4 b) { return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w); }

__global__ __launch_bounds__(kXferThreads) void copy_in_kernel(RecordParts rp, XferRecords rec, CopyInPlan pl,
                                                               const char* buf, char* wgu, char* wdn, float* ggu,
                                                               float* gdn) {
  const int row = blockIdx.y;
  const uint64_t rbytes = rp.total();
  const uint64_t step = (uint64_t)gridDim.x * kXferThreads * kXferVecPerThread;
  const uint64_t first = (uint64_t)blockIdx.x * kXferThreads * kXferVecPerThread + threadIdx.x;
  if (row < pl.n_par) {
    const int r = pl.par[row];
    const uint64_t nvec = (rp.gu_p + rp.dn_p) / 16;
    const char* src = buf + (uint64_t)r * rbytes;
    for (uint64_t v0 = first; v0 < nvec; v0 += step) {
      u32x4 a[kXferVecPerThread];
#pragma unroll
      for (int u = 0; u < kXferVecPerThread; ++u) {
        const uint64_t v = v0 + (uint64_t)u * kXferThreads;
        if (v < nvec) a[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(src + v * 16));
      }
#pragma unroll
      for (int u = 0; u < kXferVecPerThread; ++u) {
        const uint64_t v = v0 + (uint64_t)u * kXferThreads;
        if (v >= nvec) continue;
        const uint64_t off = v * 16;
        char* dst = off < rp.gu_p ? wgu + (uint64_t)rec.widx[r] * rp.gu_p + off
                                  : wdn + (uint64_t)rec.widx[r] * rp.dn_p + (off - rp.gu_p);
        __builtin_nontemporal_store(a[u], reinterpret_cast<u32x4*>(dst));
      }
    }
    return;
  }
  const int g = row - pl.n_par;
  const int tgt = pl.grp_tgt[g], start = pl.grp_start[g];
  const int a0 = pl.grp_off[g], a1 = pl.grp_off[g + 1];
  const uint64_t par_bytes = rp.gu_p + rp.dn_p;
  const uint64_t nvec = (rp.gu_g + rp.dn_g) / 16;
  const uint64_t gu_vec = rp.gu_g / 16;
  for (uint64_t v0 = first; v0 < nvec; v0 += step) {
#pragma unroll
    for (int u = 0; u < kXferVecPerThread; ++u) {
      const uint64_t v = v0 + (uint64_t)u * kXferThreads;
      if (v >= nvec) continue;
      float4* dst = v < gu_vec ? reinterpret_cast<float4*>(ggu) + (uint64_t)tgt * gu_vec + v
                               : reinterpret_cast<float4*>(gdn) + (uint64_t)tgt * (rp.dn_g / 16) + (v - gu_vec);
      float4 acc = start >= 0 ? *reinterpret_cast<const float4*>(buf + (uint64_t)start * rbytes + par_bytes + v * 16)
                              : *dst;
      for (int k = a0; k < a1; ++k)
        acc = add4(acc, *reinterpret_cast<const float4*>(buf + (uint64_t)pl.ord[k] * rbytes + par_bytes + v * 16));
      *dst = acc;
    }
  }
}

unsigned xfer_blocks_x(uint64_t nvec, int rows) {
  // about 4 workgroups per CU over all rows together
  const uint64_t per_block = (uint64_t)kXferThreads * kXferVecPerThread;
  uint64_t want = (uint64_t)num_cus() * 4 / (uint64_t)(rows > 0 ? rows : 1);
  if (want < 1) want = 1;
  const uint64_t need = (nvec + per_block - 1) / per_block;
  return (unsigned)std::max<uint64_t>(1, std::min(want, need));
}

}  // namespace
}  // namespace foremoe

using namespace foremoe;

#define REQUIRE(cond, ...)                                      \
  do {                                                          \
    if (!(cond)) return set_error(FOREMOE_EINVAL, __VA_ARGS__); \
  } while (0)

static int check_xfer_shape(const char* who, foremoe_dtype dtype, int32_t d, int32_t F, int32_t n, int32_t what) {
  REQUIRE(dtype == FOREMOE_BF16 || dtype == FOREMOE_F32, "%s: bad parameter dtype", who);
  REQUIRE(d >= 1 && F >= 1, "%s: d and F must be positive", who);
  REQUIRE(n >= 0 && n <= FOREMOE_MAX_XFER_RECORDS, "%s: n=%d outside [0, %d]", who, n, FOREMOE_MAX_XFER_RECORDS);
  REQUIRE(what >= 1 && what <= (FOREMOE_XFER_PARAMS | FOREMOE_XFER_GRADS), "%s: what=%d is not a part set", who,
          what);
  if (((int64_t)d * F) % 8 != 0)
    return set_error(FOREMOE_EUNSUPPORTED, "%s: d*F must be a multiple of 8 (16-byte record parts)", who);
  return FOREMOE_OK;
}

extern "C" {

size_t foremoe_xfer_record_bytes(int32_t d, int32_t F, foremoe_dtype dtype, int32_t what) {
  if (d < 1 || F < 1 || (dtype != FOREMOE_BF16 && dtype != FOREMOE_F32)) return 0;
  if (what < 1 || what > (FOREMOE_XFER_PARAMS | FOREMOE_XFER_GRADS)) return 0;
  return (size_t)record_parts(d, F, dtype == FOREMOE_BF16 ? 2 : 4, what).total();
}

int foremoe_copy_out(const void* w_gate_up, const void* w_down, foremoe_dtype dtype, int32_t W,
                     const float* dw_gate_up, const float* dw_down, int32_t G, int32_t d, int32_t F, int32_t n,
                     const int32_t* widx, const int32_t* gidx, int32_t what, void* buf, size_t buf_bytes,
                     void* stream) {
  int rc = check_xfer_shape("copy_out", dtype, d, F, n, what);
  if (rc) return rc;
  const RecordParts rp = record_parts(d, F, dtype == FOREMOE_BF16 ? 2 : 4, what);
  REQUIRE(buf_bytes >= (uint64_t)n * rp.total(), "copy_out: send buffer of %zu bytes, %llu needed", buf_bytes,
          (unsigned long long)((uint64_t)n * rp.total()));
  if (n == 0) return FOREMOE_OK;
  REQUIRE(buf && ((uintptr_t)buf & 15) == 0, "copy_out: send buffer NULL or not 16-byte aligned");
  XferRecords rec{};
  for (int i = 0; i < n; ++i) {
    if (what & FOREMOE_XFER_PARAMS) {
      REQUIRE(widx && widx[i] >= 0 && widx[i] < W, "copy_out: widx[%d] outside [0, W=%d)", i, W);
      rec.widx[i] = widx[i];
    }
    if (what & FOREMOE_XFER_GRADS) {
      REQUIRE(gidx && gidx[i] >= 0 && gidx[i] < G, "copy_out: gidx[%d] outside [0, G=%d)", i, G);
      rec.gidx[i] = gidx[i];
    }
  }
  REQUIRE(!(what & FOREMOE_XFER_PARAMS) || (w_gate_up && w_down), "copy_out: parameter arrays NULL");
  REQUIRE(!(what & FOREMOE_XFER_GRADS) || (dw_gate_up && dw_down), "copy_out: gradient arrays NULL");
  REQUIRE((((uintptr_t)w_gate_up | (uintptr_t)w_down | (uintptr_t)dw_gate_up | (uintptr_t)dw_down) & 15) == 0,
          "copy_out: expert arrays must be 16-byte aligned");
  const uint64_t nvec = rp.total() / 16;
  hipLaunchKernelGGL(copy_out_kernel, dim3(xfer_blocks_x(nvec, n), n), dim3(kXferThreads), 0, (hipStream_t)stream,
                     rp, rec, (const char*)w_gate_up, (const char*)w_down, (const char*)dw_gate_up,
                     (const char*)dw_down, (char*)buf);
  return check_launch("foremoe_copy_out");
}

int foremoe_copy_in(const void* buf, size_t buf_bytes, int32_t n, const int32_t* widx, const int32_t* gidx,
                    const int32_t* gmode, int32_t what, void* w_gate_up, void* w_down, foremoe_dtype dtype, int32_t W,
                    float* dw_gate_up, float* dw_down, int32_t G, int32_t d, int32_t F, void* stream) {
  int rc = check_xfer_shape("copy_in", dtype, d, F, n, what);
  if (rc) return rc;
  const RecordParts rp = record_parts(d, F, dtype == FOREMOE_BF16 ? 2 : 4, what);
  REQUIRE(buf_bytes >= (uint64_t)n * rp.total(), "copy_in: receive buffer of %zu bytes, %llu needed", buf_bytes,
          (unsigned long long)((uint64_t)n * rp.total()));
  if (n == 0) return FOREMOE_OK;
  REQUIRE(buf && ((uintptr_t)buf & 15) == 0, "copy_in: receive buffer NULL or not 16-byte aligned");
  XferRecords rec{};
  CopyInPlan pl{};
  if (what & FOREMOE_XFER_PARAMS) {
    REQUIRE(widx, "copy_in: widx is NULL");
    std::vector<char> seen(W > 0 ? W : 1, 0);
    for (int i = 0; i < n; ++i) {
      if (widx[i] < 0) continue;
      REQUIRE(widx[i] < W, "copy_in: widx[%d]=%d outside [0, W=%d)", i, widx[i], W);
      REQUIRE(!seen[widx[i]], "copy_in: two records write weight slot %d", widx[i]);
      seen[widx[i]] = 1;
      rec.widx[i] = widx[i];
      pl.par[pl.n_par++] = i;
    }
    REQUIRE(pl.n_par == 0 || (w_gate_up && w_down), "copy_in: parameter arrays NULL");
  }
  if (what & FOREMOE_XFER_GRADS) {
    REQUIRE(gidx && gmode, "copy_in: gidx or gmode is NULL");
    // gradient targets in order of first appearance; per target, start from
    // its last assign record (or its current value) and add what follows
    std::vector<int> targets;
    for (int i = 0; i < n; ++i) {
      if (gidx[i] < 0) continue;
      REQUIRE(gidx[i] < G, "copy_in: gidx[%d]=%d outside [0, G=%d)", i, gidx[i], G);
      REQUIRE(gmode[i] == FOREMOE_XFER_ASSIGN || gmode[i] == FOREMOE_XFER_ADD, "copy_in: gmode[%d]=%d", i, gmode[i]);
      if (std::find(targets.begin(), targets.end(), gidx[i]) == targets.end()) targets.push_back(gidx[i]);
    }
    int k = 0;
    for (int g : targets) {
      int start = -1;
      for (int i = 0; i < n; ++i)
        if (gidx[i] == g && gmode[i] == FOREMOE_XFER_ASSIGN) start = i;
      pl.grp_tgt[pl.n_grp] = g;
      pl.grp_start[pl.n_grp] = start;
      pl.grp_off[pl.n_grp] = k;
      for (int i = start + 1; i < n; ++i)
        if (gidx[i] == g) pl.ord[k++] = i;  // only adds follow the last assign
      ++pl.n_grp;
    }
    pl.grp_off[pl.n_grp] = k;
    REQUIRE(pl.n_grp == 0 || (dw_gate_up && dw_down), "copy_in: gradient arrays NULL");
  }
  REQUIRE((((uintptr_t)w_gate_up | (uintptr_t)w_down | (uintptr_t)dw_gate_up | (uintptr_t)dw_down) & 15) == 0,
          "copy_in: expert arrays must be 16-byte aligned");
  const int rows = pl.n_par + pl.n_grp;
  if (rows == 0) return FOREMOE_OK;
  const uint64_t nvec = std::max(rp.gu_p + rp.dn_p, rp.gu_g + rp.dn_g) / 16;
  hipLaunchKernelGGL(copy_in_kernel, dim3(xfer_blocks_x(nvec, rows), rows), dim3(kXferThreads), 0,
                     (hipStream_t)stream, rp, rec, pl, (const char*)buf, (char*)w_gate_up, (char*)w_down, dw_gate_up,
                     dw_down);
  return check_launch("foremoe_copy_in");
}

int foremoe_plan_prefetch(const int32_t* resident, int32_t W, const int32_t* needed, int32_t n, int32_t* slot_of,
                          int32_t* fetch_expert, int32_t* fetch_widx, int32_t* n_fetch) {
  REQUIRE(W >= 0 && n >= 0 && n <= W, "plan_prefetch: %d experts needed, %d weight slots", n, W);
  REQUIRE((W == 0 || resident) && (n == 0 || (needed && slot_of && fetch_expert && fetch_widx)) && n_fetch,
          "plan_prefetch: NULL array");
  // slot of each resident expert (its first slot); needed experts kept there
  std::vector<int> keep_slot(n, -1);
  std::vector<char> kept(W, 0);
  for (int i = 0; i < n; ++i) {
    REQUIRE(needed[i] >= 0, "plan_prefetch: needed[%d] < 0", i);
    for (int j = 0; j < i; ++j) REQUIRE(needed[j] != needed[i], "plan_prefetch: expert %d needed twice", needed[i]);
    for (int w = 0; w < W; ++w)
      if (resident[w] == needed[i]) {
        keep_slot[i] = w;
        kept[w] = 1;
        break;
      }
  }
  int next_free = 0, nf = 0;
  for (int i = 0; i < n; ++i) {
    if (keep_slot[i] >= 0) {
      slot_of[i] = keep_slot[i];
      continue;
    }
    while (next_free < W && kept[next_free]) ++next_free;
    if (next_free >= W) return set_error(FOREMOE_EINVAL, "plan_prefetch: more experts needed than weight slots");
    slot_of[i] = next_free;
    fetch_expert[nf] = needed[i];
    fetch_widx[nf] = next_free;
    ++nf;
    ++next_free;
  }
  *n_fetch = nf;
  return FOREMOE_OK;
}

int foremoe_prefetch_experts(const void* host_gate_up, const void* host_down, int32_t E, foremoe_dtype dtype,
                             int32_t d, int32_t F, int32_t n, const int32_t* expert, const int32_t* widx,
                             void* w_gate_up, void* w_down, int32_t W, void* stream) {
  REQUIRE(dtype == FOREMOE_BF16 || dtype == FOREMOE_F32, "prefetch_experts: bad dtype");
  REQUIRE(d >= 1 && F >= 1 && E >= 1 && W >= 1 && n >= 0 && n <= W, "prefetch_experts: bad sizes");
  if (n == 0) return FOREMOE_OK;
  REQUIRE(host_gate_up && host_down && expert && widx && w_gate_up && w_down, "prefetch_experts: NULL pointer");
  const size_t p_w = dtype == FOREMOE_BF16 ? 2 : 4;
  const size_t gu = (size_t)2 * F * d * p_w, dn = (size_t)d * F * p_w;
  for (int i = 0; i < n; ++i) {
    REQUIRE(expert[i] >= 0 && expert[i] < E, "prefetch_experts: expert[%d]=%d outside [0, E=%d)", i, expert[i], E);
    REQUIRE(widx[i] >= 0 && widx[i] < W, "prefetch_experts: widx[%d]=%d outside [0, W=%d)", i, widx[i], W);
    for (int j = 0; j < i; ++j) REQUIRE(widx[j] != widx[i], "prefetch_experts: weight slot %d written twice", widx[i]);
  }
  hipStream_t st = (hipStream_t)stream;
  for (int i = 0; i < n; ++i) {
    hipError_t e = hipMemcpyAsync((char*)w_gate_up + (size_t)widx[i] * gu,
                                  (const char*)host_gate_up + (size_t)expert[i] * gu, gu, hipMemcpyHostToDevice, st);
    if (e == hipSuccess)
      e = hipMemcpyAsync((char*)w_down + (size_t)widx[i] * dn, (const char*)host_down + (size_t)expert[i] * dn, dn,
                         hipMemcpyHostToDevice, st);
    if (e != hipSuccess) return set_error(FOREMOE_EHIP, "prefetch_experts: hipMemcpyAsync: %s", hipGetErrorString(e));
  }
  return FOREMOE_OK;
}

}  // extern "C"
