// Steps 1-3 and 5 of the per-micro-step expert layer: histogram, replica
// split, permute, combine, and the backward gathers (combine_bwd,
// permute_bwd). All integer work is exact and deterministic: per-expert
// ranks come from wavefront ballots plus prefix sums, never from the order
// in which atomics land.
#include <climits>
#include <mutex>

#include "common.h"

namespace foremoe {
namespace {

constexpr int kWaves = kHistThreads / 64;
constexpr int kPairsPerWave = kHistChunk / kWaves;

int key_bits(int E) {
  int b = 1;
  while ((1 << b) < E + 1) ++b;
  return b;
}

// Lanes of this wavefront holding the same key as this lane, restricted to
// `active`. Keys are compared bit by bit with ballots (nbits ballots).
__device__ __forceinline__ uint64_t match_key(int key, int nbits, uint64_t active) {
  uint64_t m = active;
  for (int b = 0; b < nbits; ++b) {
    const int bit = (key >> b) & 1;
    const uint64_t bal = __ballot(bit);
    m &= bit ? bal : ~bal;
  }
  return m;
}

// Key of a recorded id: the expert, -1 for padding, E for invalid ids.
__device__ __forceinline__ int id_key(int v, int E) { return v == -1 ? -1 : ((v >= 0 && v < E) ? v : E); }

// How a pair becomes its ranking key. With one source the key is the
// expert; with a per-source split (Sec. 7.2: r_{s,e,j} per source rank) it
// is s * E + e for the source s that owns the pair's token, so that ranks,
// counts and replica blocks are per (source, expert). nkeys = n_src * E is
// the invalid-id bucket.
struct KeyMap {
  int E, n_src, K;
  const int32_t* tb;  // [n_src + 1] first token of each source (n_src >= 2)
};

// Source bounds into LDS (n_src + 1 <= FOREMOE_MAX_SOURCES + 1 entries).
__device__ __forceinline__ void load_sources(const KeyMap& km, int* s_tb) {
  if (km.n_src >= 2)
    for (int i = threadIdx.x; i <= km.n_src; i += blockDim.x) s_tb[i] = km.tb[i];
}

__device__ __forceinline__ int pair_key(int v, int64_t p, const KeyMap& km, const int* s_tb) {
  const int k = id_key(v, km.E);
  if (km.n_src < 2 || k < 0) return k;
  const int nkeys = km.n_src * km.E;
  if (k == km.E) return nkeys;
  const int t = (int)(p / km.K);
  if (t < s_tb[0] || t >= s_tb[km.n_src]) return nkeys;  // token outside every source
  int lo = 0, hi = km.n_src - 1;  // the last source starting at or before t
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (s_tb[mid] <= t) lo = mid;
    else hi = mid - 1;
  }
  return lo * km.E + k;
}

// ---------------------------------------------------------------------------
// Step 1a: per-block counts of each key (bucket nkeys counts invalid ids),
// and every pair's stable rank within its block's list of the same key.
// A block's 512 pairs form 8 groups of 64 consecutive pairs, one wavefront
// each; a group's counts come from ballot key matches (no atomics), their
// prefix over the groups in pair order gives each group's base, and a
// pair's rank is its group's base plus the same-key lanes below it.
// ---------------------------------------------------------------------------
// ticket (may be NULL): the arrival ticket of the scan+split kernel that
// follows on the same stream; workgroup 0 zeroes it, so that kernel always
// starts from a zero ticket whatever the workspace held before.
constexpr int kHistIters = kHistChunk / kHistThreads;
constexpr int kHistGroups = kHistChunk / 64;
static_assert(kHistChunk % kHistThreads == 0 && kHistChunk <= 65536, "ranks are uint16 within a block");

__global__ __launch_bounds__(kHistThreads) void hist_count_kernel(const int32_t* __restrict__ ids, int64_t npairs,
                                                                  KeyMap km, int E, int nbits,
                                                                  int32_t* __restrict__ partial,
                                                                  uint16_t* __restrict__ rank, uint32_t* ticket) {
  __shared__ int s_g[kHistGroups][FOREMOE_MAX_EXPERTS + 1];
  __shared__ int s_tb[FOREMOE_MAX_SOURCES + 1];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  if (ticket && blockIdx.x == 0 && tid == 0) atomicExch(ticket, 0u);
  for (int i = tid; i < kHistGroups * (E + 1); i += kHistThreads) s_g[i / (E + 1)][i % (E + 1)] = 0;
  load_sources(km, s_tb);
  __syncthreads();
  const int64_t base = (int64_t)blockIdx.x * kHistChunk;
  int key[kHistIters];
  uint64_t m[kHistIters];
#pragma unroll
  for (int i = 0; i < kHistIters; ++i) {
    // group i * kWaves + w holds pairs base + (i * kWaves + w) * 64 + lane
    const int64_t p = base + (int64_t)i * kHistThreads + tid;
    key[i] = -1;
    if (p < npairs) key[i] = pair_key(ids[p], p, km, s_tb);
    const uint64_t active = __ballot(key[i] >= 0);
    m[i] = match_key(key[i], nbits, active);
    if (key[i] >= 0 && lane == __builtin_ctzll(m[i])) s_g[i * kWaves + w][key[i]] = __popcll(m[i]);
  }
  __syncthreads();
  int32_t* out = partial + (int64_t)blockIdx.x * (E + 1);
  for (int e = tid; e <= E; e += kHistThreads) {
    int run = 0;
#pragma unroll
    for (int g = 0; g < kHistGroups; ++g) {
      const int c = s_g[g][e];
      s_g[g][e] = run;
      run += c;
    }
    out[e] = run;
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < kHistIters; ++i) {
    const int64_t p = base + (int64_t)i * kHistThreads + tid;
    if (p < npairs)
      rank[p] = (uint16_t)((key[i] >= 0 && key[i] < E) ? s_g[i * kWaves + w][key[i]] + lanes_below(m[i]) : 0);
  }
}

// Inclusive block-wide scan of one int per thread (NW wavefronts).
template <int NW = kWaves>
__device__ int block_inclusive_scan(int v, int* s_tmp /* [NW] */, int& total) {
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
  for (int i = 0; i < NW; ++i) {
    const int t = s_tmp[i];
    if (i < w) before += t;
    total += t;
  }
  __syncthreads();
  return v + before;
}

// ---------------------------------------------------------------------------
// Step 1b: for each expert (one workgroup per expert column) turn the
// per-block counts into exclusive block bases; the total is counts[e]
// (bucket E: the invalid-id count status word).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kHistThreads) void hist_scan_kernel(int32_t* __restrict__ partial, int64_t nblocks, int E,
                                                                 int32_t* __restrict__ counts, int32_t* __restrict__ status) {
  __shared__ int s_tmp[kWaves];
  const int e = blockIdx.x;
  int carry = 0;
  for (int64_t b0 = 0; b0 < nblocks; b0 += kHistThreads) {
    const int64_t b = b0 + threadIdx.x;
    const int v = b < nblocks ? partial[b * (E + 1) + e] : 0;
    int total;
    const int incl = block_inclusive_scan(v, s_tmp, total);
    if (b < nblocks) partial[b * (E + 1) + e] = carry + incl - v;
    carry += total;
  }
  if (threadIdx.x == 0) {
    if (e < E) counts[e] = carry;
    else status[FOREMOE_WS_INVALID_IDS] = carry;
  }
}

// ---------------------------------------------------------------------------
// Step 2: replica boundaries, slot counts and slot offsets (one workgroup).
// ---------------------------------------------------------------------------
struct PlanDev {
  int E, S, R_max, n_src;  // n_src >= 1
  const int32_t* slot_expert;
  const int32_t* slot_replica;
  const int32_t* expert_nrep;
  const int32_t* expert_rep_weight;
  const int32_t* src_rep_weight;  // [n_src * E * R_max] or NULL
};

__device__ __forceinline__ int clamp_nrep(const PlanDev& P, int e, int& err) {
  int R = P.expert_nrep[e];
  if (R < 1 || R > P.R_max) {
    ++err;
    R = 1;
  }
  return R;
}

// Keys are (source, expert) pairs kk = s * E + e and the S slots are split
// into virtual slots jj = j * n_src + s (one source: kk = e, jj = j).
// Virtual slot jj takes replica r_j of key s * E + e_j; its rows follow
// those of the same slot's earlier sources, so a slot's rows are its
// sources' blocks in source order. One workgroup of 1024 threads keeps the
// replica bounds and the replica -> slot table in LDS while it works, loads
// each key's weights together, and writes both tables out at the end, so
// the kernel costs a few memory round trips.
// Two sizes: up to 256 keys with 256 threads (small LDS, quick to launch)
// and up to FOREMOE_MAX_EXPERTS keys with 1024 threads.
// `counts` may point to global memory or to LDS.
template <int kAssignThreads, int MAXK>
__device__ __forceinline__ void assign_block(const int32_t* counts, const PlanDev& P, int32_t* __restrict__ rep_begin,
                                             int32_t* __restrict__ slot_count, int32_t* __restrict__ slot_offset,
                                             int32_t* __restrict__ vslot_offset, int32_t* __restrict__ rep_slot,
                                             int32_t* __restrict__ status) {
  constexpr int NW = kAssignThreads / 64;
  __shared__ int s_err;
  __shared__ int s_nrep[FOREMOE_MAX_EXPERTS];
  __shared__ int s_rs[MAXK * FOREMOE_MAX_REPLICAS];
  __shared__ int s_rb[MAXK * (FOREMOE_MAX_REPLICAS + 1)];
  __shared__ int s_cnt[FOREMOE_MAX_SLOTS];
  __shared__ int s_off[FOREMOE_MAX_SLOTS + 1];
  __shared__ int s_tmp[NW];
  const int tid = threadIdx.x;
  if (tid == 0) s_err = 0;
  const int RS = P.R_max + 1;
  const int NK = P.n_src * P.E, NS = P.n_src * P.S;
  int err = 0;
  for (int e = tid; e < P.E; e += kAssignThreads) s_nrep[e] = clamp_nrep(P, e, err);
  for (int i = tid; i < NK * P.R_max; i += kAssignThreads) s_rs[i] = INT_MAX;
  __syncthreads();
  for (int kk = tid; kk < NK; kk += kAssignThreads) {
    const int e = kk % P.E;
    const int n = counts[kk];
    const int R = s_nrep[e];
    const int32_t* wt = P.src_rep_weight ? P.src_rep_weight + (int64_t)kk * P.R_max
                                          : (P.expert_rep_weight ? P.expert_rep_weight + (int64_t)e * P.R_max : nullptr);
    int wv[FOREMOE_MAX_REPLICAS];
#pragma unroll
    for (int r = 0; r < FOREMOE_MAX_REPLICAS; ++r) wv[r] = (r < R) ? (wt ? wt[r] : 1) : 0;
    long long total = 0;
    bool bad = false;
#pragma unroll
    for (int r = 0; r < FOREMOE_MAX_REPLICAS; ++r) {
      if (wv[r] < 0) bad = true;
      total += wv[r];
    }
    // all-zero per-source weights are fine for an empty block
    if (total <= 0 && (n > 0 || !P.src_rep_weight)) bad = true;
    if (bad) ++err;
    const bool eq = bad || total <= 0;
    const long long den = eq ? (long long)R : total;
    long long pref = 0;
    int* rb = s_rb + kk * RS;
    rb[0] = 0;
    for (int r = 0; r < P.R_max; ++r) {
      if (r < R) {
        pref += eq ? 1 : wv[r];
        rb[r + 1] = (int)(((long long)n * pref) / den);
      } else {
        rb[r + 1] = n;
      }
    }
  }
  // Virtual slot jj claims replica (key, r); with duplicates the lowest slot wins.
  for (int jj = tid; jj < NS; jj += kAssignThreads) {
    const int j = jj / P.n_src, src = jj % P.n_src;
    const int e = P.slot_expert[j], r = P.slot_replica[j];
    if (e >= 0 && e < P.E && r >= 0 && r < P.R_max) atomicMin(&s_rs[(src * P.E + e) * P.R_max + r], jj);
  }
  __syncthreads();
  for (int i = tid; i < NK * RS; i += kAssignThreads) rep_begin[i] = s_rb[i];
  for (int jj = tid; jj < NS; jj += kAssignThreads) {
    const int j = jj / P.n_src, src = jj % P.n_src;
    const int e = P.slot_expert[j], r = P.slot_replica[j];
    int c = 0;
    bool ok = false;
    if (e >= 0 && e < P.E && r >= 0 && r < s_nrep[e]) {
      const int kk = src * P.E + e;
      if (s_rs[kk * P.R_max + r] == jj) {
        c = s_rb[kk * RS + r + 1] - s_rb[kk * RS + r];
        ok = true;
      }
    }
    if (!ok && src == 0) ++err;  // one error per bad slot
    s_cnt[jj] = c;
  }
  if (err) atomicAdd(&s_err, err);
  for (int i = tid; i < NK * P.R_max; i += kAssignThreads) {
    // replicas beyond R_e, and replicas held by no (valid) slot, are remote
    const int e = (i / P.R_max) % P.E, r = i % P.R_max;
    const int v = s_rs[i];
    rep_slot[i] = (v == INT_MAX || r >= s_nrep[e]) ? -1 : v;
  }
  __syncthreads();
  int carry = 0;
  for (int j0 = 0; j0 < NS; j0 += kAssignThreads) {
    const int jj = j0 + tid;
    const int v = jj < NS ? s_cnt[jj] : 0;
    int total;
    const int incl = block_inclusive_scan<NW>(v, s_tmp, total);
    if (jj < NS) s_off[jj] = carry + incl - v;
    carry += total;
  }
  if (tid == 0) s_off[NS] = carry;
  __syncthreads();
  for (int jj = tid; jj <= NS; jj += kAssignThreads) vslot_offset[jj] = s_off[jj];
  for (int j = tid; j < P.S; j += kAssignThreads) {
    int c = 0;
    for (int src = 0; src < P.n_src; ++src) c += s_cnt[j * P.n_src + src];
    slot_count[j] = c;
    slot_offset[j] = s_off[j * P.n_src];
  }
  if (tid == 0) {
    slot_offset[P.S] = carry;
    status[FOREMOE_WS_PLAN_ERRORS] = s_err;
  }
}

template <int kAssignThreads, int MAXK>
__global__ __launch_bounds__(kAssignThreads) void assign_kernel(const int32_t* __restrict__ counts, PlanDev P,
                                                                int32_t* __restrict__ rep_begin, int32_t* __restrict__ slot_count,
                                                                int32_t* __restrict__ slot_offset, int32_t* __restrict__ vslot_offset,
                                                                int32_t* __restrict__ rep_slot, int32_t* __restrict__ status) {
  assign_block<kAssignThreads, MAXK>(counts, P, rep_begin, slot_count, slot_offset, vslot_offset, rep_slot, status);
}

// ---------------------------------------------------------------------------
// Step 1b and step 2 in one launch (up to 256 keys): one workgroup per key
// column turns the per-block counts into block bases and the key's total,
// as hist_scan_kernel does; the last workgroup to finish (a ticket in the
// workspace header) then splits the keys over the replicas, as
// assign_kernel does. Workgroups may run on different XCDs, whose L2
// caches are not coherent with each other: the totals are stored and loaded
// with device scope (SC1 cache policy: written through, never read from a
// stale line), and each workgroup's total has reached memory before it
// takes its ticket (its block bases, read only by later kernels, are stored
// after). No workgroup waits for another. The ticket is zero on entry: the
// count kernel before it on the same stream has zeroed it.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kHistThreads) void hist_scan_assign_kernel(
    int32_t* __restrict__ partial, int64_t nblocks, int nkeys, int32_t* __restrict__ counts, uint32_t* ticket,
    PlanDev P, int32_t* __restrict__ rep_begin, int32_t* __restrict__ slot_count, int32_t* __restrict__ slot_offset,
    int32_t* __restrict__ vslot_offset, int32_t* __restrict__ rep_slot, int32_t* __restrict__ status) {
  __shared__ int s_tmp[kWaves];
  __shared__ int s_cnt[257];
  __shared__ int s_last;
  // the plan's tables (at most 256 keys here), loaded by every workgroup
  // beside its column so that the last one finds them in LDS
  __shared__ int s_nrep[256];
  __shared__ int s_w[256 * FOREMOE_MAX_REPLICAS];
  __shared__ int s_se[FOREMOE_MAX_SLOTS];
  __shared__ int s_sr[FOREMOE_MAX_SLOTS];
  const int e = blockIdx.x, tid = threadIdx.x;
  const int v_first = tid < nblocks ? partial[(int64_t)tid * (nkeys + 1) + e] : 0;
  const int32_t* wsrc = P.src_rep_weight ? P.src_rep_weight : P.expert_rep_weight;
  const int nw = P.src_rep_weight ? nkeys * P.R_max : (P.expert_rep_weight ? P.E * P.R_max : 0);
  for (int i = tid; i < P.E; i += kHistThreads) s_nrep[i] = P.expert_nrep[i];
  for (int i = tid; i < nw; i += kHistThreads) s_w[i] = wsrc[i];
  for (int i = tid; i < P.S; i += kHistThreads) {
    s_se[i] = P.slot_expert[i];
    s_sr[i] = P.slot_replica[i];
  }
  // one chunk of blocks (the usual case): the block bases are stored after
  // the ticket, so that taking it waits only for the total's store
  const bool defer = nblocks <= kHistThreads;
  int base_first = 0;
  int carry = 0;
  for (int64_t b0 = 0; b0 < nblocks; b0 += kHistThreads) {
    const int64_t b = b0 + tid;
    const int v = b0 == 0 ? v_first : (b < nblocks ? partial[b * (nkeys + 1) + e] : 0);
    int total;
    const int incl = block_inclusive_scan(v, s_tmp, total);
    if (b < nblocks) {
      if (defer) base_first = carry + incl - v;
      else partial[b * (nkeys + 1) + e] = carry + incl - v;
    }
    carry += total;
  }
  if (tid == 0) {
    if (e < nkeys) __hip_atomic_store(counts + e, carry, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    else status[FOREMOE_WS_INVALID_IDS] = carry;
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): the total has reached memory
    s_last = atomicAdd(ticket, 1u) == gridDim.x - 1;
  }
  __syncthreads();
  if (defer && tid < nblocks) partial[(int64_t)tid * (nkeys + 1) + e] = base_first;
  if (!s_last) return;
  for (int k = tid; k < nkeys; k += kHistThreads)
    s_cnt[k] = __hip_atomic_load(counts + k, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  PlanDev L = P;
  L.expert_nrep = s_nrep;
  L.slot_expert = s_se;
  L.slot_replica = s_sr;
  if (P.src_rep_weight) L.src_rep_weight = s_w;
  else if (P.expert_rep_weight) L.expert_rep_weight = s_w;
  assign_block<kHistThreads, 256>(s_cnt, L, rep_begin, slot_count, slot_offset, vslot_offset, rep_slot, status);
  if (tid == 0) atomicExch(ticket, 0u);  // ready for the next call
}

// ---------------------------------------------------------------------------
// Step 3: rank, replica, slot and row of every pair, both index maps, and
// the rows of x gathered into slot order, in one pass over the pairs. A
// wavefront takes 64 consecutive pairs, one per lane: a pair's rank in its
// key's list is its block's base (the scanned partial counts) plus its rank
// within the block (written by the count kernel). The wavefront then copies
// the rows of its local pairs, kRowsPerWave at a time: every 16-byte load of
// a group is issued before its stores. A group is shared by nsub * ncol
// wavefronts, each of which finds the group's rows (the first writes the
// index maps): with few pairs (fewer groups of 64 than 16 wavefronts per
// CU) wavefront s of nsub copies the local pairs whose index among the
// group's local pairs is s modulo nsub; with rows wider than one copy pass
// (64 * kVecPerLane vectors), wavefront c of ncol copies passes c, c +
// ncol, ... of each of its rows, so that no wavefront waits for the loads
// of one pass before issuing the next (with every wavefront in step, all
// of them would read, then all write, and the two would not overlap).
// ---------------------------------------------------------------------------
constexpr int kRowsPerWave = 4;
constexpr int kVecPerLane = 4;  // 16-byte vectors per lane per row and pass

// Range-checked 16-byte loads from one wave-uniform byte range: offsets at or
// past `bytes` read as zero without touching memory, so loads need no branch
// (and a zero-byte range turns a whole row of loads into zeros).
struct RowReader {
  __amdgpu_buffer_rsrc_t rs;
  __device__ __forceinline__ RowReader(const void* base, uint32_t bytes)
      : rs(__builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000)) {}
  __device__ __forceinline__ uint4 load(uint32_t off) const {
    const auto v = __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0);
    return make_uint4(v[0], v[1], v[2], v[3]);
  }
};

__global__ __launch_bounds__(256) void permute_gather_kernel(
    const uint4* __restrict__ x, int64_t vec_per_row, const int32_t* __restrict__ ids, int64_t npairs, KeyMap km,
    int nkeys, int R_max, const int32_t* __restrict__ block_base, const uint16_t* __restrict__ rank,
    const int32_t* __restrict__ rep_begin, const int32_t* __restrict__ rep_slot, const int32_t* __restrict__ row_off,
    int S, const int32_t* __restrict__ n_rows_dev, int64_t n_cap, int32_t* __restrict__ pair_to_row,
    int32_t* __restrict__ row_to_pair, uint4* __restrict__ x_perm, int32_t* __restrict__ status, int nsub,
    int ncol) {
  __shared__ int s_tb[FOREMOE_MAX_SOURCES + 1];
  load_sources(km, s_tb);
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int64_t wave = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int64_t nwaves = (int64_t)gridDim.x * 4;
  const int RS = R_max + 1;
  const uint32_t row_bytes = (uint32_t)(vec_per_row * 16);
  const int64_t ngroups = (npairs + 63) / 64;
  const int per = nsub * ncol;  // wavefronts per group
  for (int64_t W = wave; W < ngroups * per; W += nwaves) {
    const int64_t g = W / per;
    const int sub = (int)(W % per) / ncol, col = (int)(W % per) % ncol;
    const int64_t p = g * 64 + lane;
    int row = -1, tok = -1;
    if (p < npairs) {
      const int key = pair_key(ids[p], p, km, s_tb);
      if (key >= 0 && key < nkeys) {
        const int q = block_base[(p / kHistChunk) * (nkeys + 1) + key] + (int)rank[p];
        const int32_t* rb = rep_begin + (int64_t)key * RS;
        int r = 0;
        while (r + 1 < R_max && rb[r + 1] <= q) ++r;
        const int j = rep_slot[key * R_max + r];
        if (j >= 0 && j < S) {
          const int64_t rr = (int64_t)row_off[j] + q - rb[r];
          if (rr >= 0 && rr < n_cap) {
            row = (int)rr;
            tok = (int)(p / km.K);
            if (sub == 0 && col == 0) row_to_pair[row] = (int32_t)p;
          }
        }
      }
      if (sub == 0 && col == 0) pair_to_row[p] = row;
    }
    // this wavefront's share of the group's local pairs
    const uint64_t all = __ballot(row >= 0);
    uint64_t local = __ballot(row >= 0 && lanes_below(all) % nsub == sub);
    while (local) {
      int rows[kRowsPerWave], toks[kRowsPerWave];
#pragma unroll
      for (int r = 0; r < kRowsPerWave; ++r) {
        rows[r] = -1;
        toks[r] = -1;
        if (local) {
          const int l = __builtin_ctzll(local);
          local &= local - 1;
          rows[r] = __builtin_amdgcn_readlane(row, l);
          toks[r] = __builtin_amdgcn_readlane(tok, l);
        }
      }
      // a token's local pairs are consecutive lanes: a row of the group whose
      // token equals the one before it is loaded once and stored twice
      bool dup[kRowsPerWave];
#pragma unroll
      for (int r = 0; r < kRowsPerWave; ++r) dup[r] = r > 0 && toks[r] >= 0 && toks[r] == toks[r - 1];
      for (int64_t v0 = (int64_t)col * 64 * kVecPerLane; v0 < vec_per_row; v0 += (int64_t)ncol * 64 * kVecPerLane) {
        uint4 a[kRowsPerWave][kVecPerLane];
#pragma unroll
        for (int r = 0; r < kRowsPerWave; ++r) {
          const bool ld = toks[r] >= 0 && !dup[r];
          const RowReader rd(ld ? (const void*)(x + (int64_t)toks[r] * vec_per_row) : (const void*)x,
                             ld ? row_bytes : 0u);
#pragma unroll
          for (int u = 0; u < kVecPerLane; ++u) a[r][u] = rd.load((uint32_t)((v0 + u * 64 + lane) * 16));
        }
#pragma unroll
        for (int r = 1; r < kRowsPerWave; ++r) {
          if (dup[r]) {
#pragma unroll
            for (int u = 0; u < kVecPerLane; ++u) a[r][u] = a[r - 1][u];
          }
        }
#pragma unroll
        for (int r = 0; r < kRowsPerWave; ++r) {
          if (rows[r] < 0) continue;
#pragma unroll
          for (int u = 0; u < kVecPerLane; ++u) {
            const int64_t vi = v0 + u * 64 + lane;
            if (vi < vec_per_row) x_perm[(int64_t)rows[r] * vec_per_row + vi] = a[r][u];
          }
        }
      }
    }
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    const int64_t N = *n_rows_dev;
    status[FOREMOE_WS_DROPPED] = N > n_cap ? (int)(N - n_cap) : 0;
  }
}

// ---------------------------------------------------------------------------
// Vector helpers for the gathers: one "vector" is 16 bytes of input
// (8 bf16 or 4 fp32), widened to floats.
// ---------------------------------------------------------------------------
template <typename T>
struct Vec;

template <>
struct Vec<uint16_t> {
  static constexpr int N = 8;
  __device__ static void widen(const uint4& v, float* f) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f[2 * i] = bf2f(w[i] & 0xFFFFu);
      f[2 * i + 1] = bf2f(w[i] >> 16);
    }
  }
  template <int M>
  __device__ static void store(uint16_t* p, const float* f) {
    static_assert(M % 2 == 0, "even element count");
    uint32_t w[M / 2];
#pragma unroll
    for (int i = 0; i < M / 2; ++i) w[i] = pack_bf2(f[2 * i], f[2 * i + 1]);
    if constexpr (M == 8) {
      *reinterpret_cast<uint4*>(p) = make_uint4(w[0], w[1], w[2], w[3]);
    } else {
      *reinterpret_cast<uint2*>(p) = make_uint2(w[0], w[1]);
    }
  }
};

template <>
struct Vec<float> {
  static constexpr int N = 4;
  __device__ static void widen(const uint4& v, float* f) {
    f[0] = __uint_as_float(v.x);
    f[1] = __uint_as_float(v.y);
    f[2] = __uint_as_float(v.z);
    f[3] = __uint_as_float(v.w);
  }
  template <int M>
  __device__ static void store(float* p, const float* f) {
#pragma unroll
    for (int i = 0; i < M; i += 4) *reinterpret_cast<float4*>(p + i) = make_float4(f[i], f[i + 1], f[i + 2], f[i + 3]);
  }
};

constexpr int kGatherChunk = 2;  // 16-byte vectors per lane per pass
constexpr int kPairGroup = 4;    // pairs of a token whose rows are loaded together

// The row and gate of the token's pairs: lane k < K holds pair k; `valid`
// has bit k set when that pair was computed here.
struct TokenPairs {
  int row;
  float gate;
  uint64_t valid;
};

__device__ __forceinline__ TokenPairs token_pairs(const int32_t* __restrict__ pair_to_row,
                                                  const float* __restrict__ gates, int64_t t, int K, int64_t n_cap) {
  // K <= FOREMOE_MAX_TOPK = 64: one lane per pair
  const int lane = threadIdx.x & 63;
  TokenPairs tp;
  tp.row = -1;
  tp.gate = 1.0f;
  const int k = lane;
  if (k < K) {
    const int r = pair_to_row[t * K + k];
    if (r >= 0 && r < n_cap) tp.row = r;
    if (gates) tp.gate = gates[t * K + k];
  }
  tp.valid = __ballot(tp.row >= 0);
  return tp;
}

// ---------------------------------------------------------------------------
// Step 5 (and the backward of step 3 with unit weights): one wavefront per
// token, y[t] = sum_k g_k * Y[row_k] in ascending k, fp32 accumulation. The
// rows of up to kPairGroup pairs are loaded together before accumulating.
// ---------------------------------------------------------------------------
template <typename Tin, typename Tout>
__global__ __launch_bounds__(256) void combine_kernel(const Tin* __restrict__ y_perm, const int32_t* __restrict__ pair_to_row,
                                                      const float* __restrict__ gates, int64_t T, int K, int d,
                                                      int64_t n_cap, Tout* __restrict__ y) {
  constexpr int VE = Vec<Tin>::N;
  const int lane = threadIdx.x & 63;
  const int64_t wave = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int64_t nwaves = (int64_t)gridDim.x * 4;
  const int nvec = d / VE;
  const uint32_t row_bytes = (uint32_t)d * (uint32_t)sizeof(Tin);
  for (int64_t t = wave; t < T; t += nwaves) {
    const TokenPairs tp = token_pairs(pair_to_row, gates, t, K, n_cap);
    for (int v0 = 0; v0 < nvec; v0 += 64 * kGatherChunk) {
      float acc[kGatherChunk][VE];
#pragma unroll
      for (int u = 0; u < kGatherChunk; ++u)
#pragma unroll
        for (int i = 0; i < VE; ++i) acc[u][i] = 0.f;
      uint64_t m = tp.valid;
      while (m) {
        int ks[kPairGroup];
        int n = 0;
#pragma unroll
        for (int q = 0; q < kPairGroup; ++q) {
          ks[q] = m ? __builtin_ctzll(m) : -1;
          if (m) {
            m &= m - 1;
            ++n;
          }
        }
        uint4 raw[kPairGroup][kGatherChunk];
#pragma unroll
        for (int q = 0; q < kPairGroup; ++q) {
          const int row = __builtin_amdgcn_readfirstlane(q < n ? __shfl(tp.row, ks[q], 64) : 0);
          const RowReader rd(y_perm + (int64_t)row * d, q < n ? row_bytes : 0u);
#pragma unroll
          for (int u = 0; u < kGatherChunk; ++u) raw[q][u] = rd.load((uint32_t)((v0 + u * 64 + lane) * 16));
        }
#pragma unroll
        for (int q = 0; q < kPairGroup; ++q) {
          if (q >= n) break;
          const float g = __shfl(tp.gate, ks[q], 64);
#pragma unroll
          for (int u = 0; u < kGatherChunk; ++u) {
            float v[VE];
            Vec<Tin>::widen(raw[q][u], v);
#pragma unroll
            for (int i = 0; i < VE; ++i) acc[u][i] += g * v[i];
          }
        }
      }
      Tout* dst = y + t * d;
#pragma unroll
      for (int u = 0; u < kGatherChunk; ++u) {
        const int vi = v0 + u * 64 + lane;
        if (vi < nvec) Vec<Tout>::template store<VE>(dst + (int64_t)vi * VE, acc[u]);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Backward of step 5: one wavefront per token; for each local pair write
// dY[row] = g * dy[t] and dgates[p] = <dy[t], Y[row]> (fixed-order butterfly
// and chunk sums); dgates of non-local pairs = 0. dy[t] is loaded once per
// column chunk, the rows of up to kPairGroup pairs together.
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void combine_bwd_kernel(const T* __restrict__ dy, const T* __restrict__ y_perm,
                                                          const int32_t* __restrict__ pair_to_row,
                                                          const float* __restrict__ gates, int64_t Ttok, int K, int d,
                                                          int64_t n_cap, T* __restrict__ dy_perm, float* __restrict__ dgates) {
  constexpr int VE = Vec<T>::N;
  const int lane = threadIdx.x & 63;
  const int64_t wave = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int64_t nwaves = (int64_t)gridDim.x * 4;
  const int nvec = d / VE;
  const uint32_t row_bytes = (uint32_t)d * (uint32_t)sizeof(T);
  for (int64_t t = wave; t < Ttok; t += nwaves) {
    const T* dyt = dy + t * d;
    {
      const TokenPairs tp = token_pairs(pair_to_row, gates, t, K, n_cap);
      // pairs not computed here get a zero gate gradient
      if (dgates && lane < K && tp.row < 0) dgates[t * K + lane] = 0.f;
      uint64_t m = tp.valid;
      while (m) {
        int ks[kPairGroup];
        int n = 0;
#pragma unroll
        for (int q = 0; q < kPairGroup; ++q) {
          ks[q] = m ? __builtin_ctzll(m) : -1;
          if (m) {
            m &= m - 1;
            ++n;
          }
        }
        int rows[kPairGroup];
        float gs[kPairGroup], part[kPairGroup];
#pragma unroll
        for (int q = 0; q < kPairGroup; ++q) {
          rows[q] = __builtin_amdgcn_readfirstlane(q < n ? __shfl(tp.row, ks[q], 64) : 0);
          gs[q] = q < n ? __shfl(tp.gate, ks[q], 64) : 0.f;
          part[q] = 0.f;
        }
        const RowReader rdy(dyt, row_bytes);
        for (int v0 = 0; v0 < nvec; v0 += 64 * kGatherChunk) {
          uint4 ra[kGatherChunk];
          uint4 rb[kPairGroup][kGatherChunk];
#pragma unroll
          for (int u = 0; u < kGatherChunk; ++u) ra[u] = rdy.load((uint32_t)((v0 + u * 64 + lane) * 16));
#pragma unroll
          for (int q = 0; q < kPairGroup; ++q) {
            const RowReader rd(y_perm + (int64_t)rows[q] * d, (dgates && q < n) ? row_bytes : 0u);
#pragma unroll
            for (int u = 0; u < kGatherChunk; ++u) rb[q][u] = rd.load((uint32_t)((v0 + u * 64 + lane) * 16));
          }
#pragma unroll
          for (int q = 0; q < kPairGroup; ++q) {
            if (q >= n) break;
#pragma unroll
            for (int u = 0; u < kGatherChunk; ++u) {
              const int vi = v0 + u * 64 + lane;
              float a[VE], b[VE], o[VE];
              Vec<T>::widen(ra[u], a);
              Vec<T>::widen(rb[q][u], b);
#pragma unroll
              for (int i = 0; i < VE; ++i) {
                o[i] = gs[q] * a[i];
                part[q] += a[i] * b[i];
              }
              if (vi < nvec) Vec<T>::template store<VE>(dy_perm + (int64_t)rows[q] * d + (int64_t)vi * VE, o);
            }
          }
        }
        if (dgates) {
#pragma unroll
          for (int q = 0; q < kPairGroup; ++q) {
            if (q >= n) break;
            const float s = wave_sum(part[q]);
            if (lane == 0) dgates[t * K + ks[q]] = s;
          }
        }
      }
    }
  }
}

int gather_grid(int64_t items) {
  // four wavefronts per workgroup; enough workgroups to fill the chip
  int64_t blocks = (items + 3) / 4;
  const int64_t cap = (int64_t)num_cus() * 16;
  if (blocks > cap) blocks = cap;
  if (blocks < 1) blocks = 1;
  return (int)blocks;
}

}  // namespace
}  // namespace foremoe

using namespace foremoe;

#define REQUIRE(cond, ...)                                      \
  do {                                                          \
    if (!(cond)) return set_error(FOREMOE_EINVAL, __VA_ARGS__); \
  } while (0)

extern "C" {

static int check_hist(const char* who, const int32_t* ids, int64_t T, int32_t K, int32_t E, const int32_t* counts,
                      const void* ws, size_t ws_bytes) {
  REQUIRE(T >= 0, "%s: T < 0", who);
  REQUIRE(K >= 1 && K <= FOREMOE_MAX_TOPK, "%s: K=%d outside [1, %d]", who, K, FOREMOE_MAX_TOPK);
  REQUIRE(E >= 1 && E <= FOREMOE_MAX_EXPERTS, "%s: %d keys outside [1, %d]", who, E, FOREMOE_MAX_EXPERTS);
  REQUIRE(T * (int64_t)K < (int64_t)INT_MAX, "%s: T*K must be below 2^31", who);
  REQUIRE(ids || T == 0, "%s: ids is NULL", who);
  REQUIRE(counts && ws, "%s: counts or ws is NULL", who);
  REQUIRE(ws_bytes >= ws_bytes_needed(T, K, E), "%s: workspace too small (%zu < %zu)", who, ws_bytes,
          ws_bytes_needed(T, K, E));
  return FOREMOE_OK;
}

// status: where the status words go (the workspace header, or a caller's
// array in foremoe_dispatch_static).
static int histogram_common(const char* who, const int32_t* ids, int64_t T, int32_t K, int32_t E, KeyMap km,
                            int32_t* counts, void* ws, size_t ws_bytes, int32_t* status, void* stream) {
  int rc = check_hist(who, ids, T, K, E, counts, ws, ws_bytes);
  if (rc) return rc;
  hipStream_t st = (hipStream_t)stream;
  const int64_t npairs = T * (int64_t)K;
  const int64_t nb = hist_blocks(npairs);
  int32_t* partial = (int32_t*)((char*)ws + kWsPartialOff);
  uint16_t* rank = (uint16_t*)((char*)ws + ws_rank_off(T, K, E));
  hipLaunchKernelGGL(hist_count_kernel, dim3((unsigned)nb), dim3(kHistThreads), 0, st, ids, npairs, km, E,
                     key_bits(E), partial, rank, (uint32_t*)nullptr);
  hipLaunchKernelGGL(hist_scan_kernel, dim3(E + 1), dim3(kHistThreads), 0, st, partial, nb, E, counts, status);
  return check_launch(who);
}

int foremoe_histogram(const int32_t* ids, int64_t T, int32_t K, int32_t E, int32_t* counts, void* ws,
                      size_t ws_bytes, void* stream) {
  return histogram_common("foremoe_histogram", ids, T, K, E, KeyMap{E, 1, K, nullptr}, counts, ws, ws_bytes,
                          (int32_t*)ws, stream);
}

int foremoe_histogram_src(const int32_t* ids, int64_t T, int32_t K, int32_t E, int32_t n_src,
                          const int32_t* src_token_begin, int32_t* counts, void* ws, size_t ws_bytes, void* stream) {
  REQUIRE(n_src >= 2 && n_src <= FOREMOE_MAX_SOURCES, "histogram_src: n_src=%d outside [2, %d]", n_src,
          FOREMOE_MAX_SOURCES);
  REQUIRE(E >= 1 && (int64_t)E * n_src <= FOREMOE_MAX_EXPERTS, "histogram_src: n_src * E must be in [1, %d]",
          FOREMOE_MAX_EXPERTS);
  REQUIRE(src_token_begin, "histogram_src: src_token_begin is NULL");
  return histogram_common("foremoe_histogram_src", ids, T, K, E * n_src, KeyMap{E, n_src, K, src_token_begin},
                          counts, ws, ws_bytes, (int32_t*)ws, stream);
}

static int check_plan(const foremoe_plan* plan, const int32_t* counts, const int32_t* rep_begin,
                      const int32_t* slot_count, const int32_t* slot_offset, const void* ws, size_t ws_bytes) {
  REQUIRE(plan, "assign_replicas: plan is NULL");
  REQUIRE(plan->E >= 1 && plan->E <= FOREMOE_MAX_EXPERTS, "assign_replicas: E=%d out of range", plan->E);
  REQUIRE(plan->S >= 0 && plan->S <= FOREMOE_MAX_SLOTS, "assign_replicas: S=%d out of range", plan->S);
  REQUIRE(plan->R_max >= 1 && plan->R_max <= FOREMOE_MAX_REPLICAS, "assign_replicas: R_max=%d out of range",
          plan->R_max);
  REQUIRE(counts && rep_begin && slot_offset && ws, "assign_replicas: NULL buffer");
  REQUIRE(plan->expert_nrep, "assign_replicas: plan->expert_nrep is NULL");
  REQUIRE(plan->S == 0 || (plan->slot_expert && plan->slot_replica && slot_count),
          "assign_replicas: NULL slot arrays");
  REQUIRE(ws_bytes >= kWsPartialOff, "assign_replicas: workspace too small");
  const int n_src = plan->n_src < 1 ? 1 : plan->n_src;
  if (n_src >= 2) {
    REQUIRE(n_src <= FOREMOE_MAX_SOURCES, "assign_replicas: n_src=%d above %d", n_src, FOREMOE_MAX_SOURCES);
    REQUIRE((int64_t)n_src * plan->E <= FOREMOE_MAX_EXPERTS && (int64_t)n_src * plan->S <= FOREMOE_MAX_SLOTS,
            "assign_replicas: n_src * E or n_src * S above the limits");
    REQUIRE(plan->src_token_begin, "assign_replicas: plan->src_token_begin is NULL");
  }
  return FOREMOE_OK;
}

static PlanDev plan_dev(const foremoe_plan* plan) {
  const int n_src = plan->n_src < 1 ? 1 : plan->n_src;
  return PlanDev{plan->E, plan->S, plan->R_max, n_src, plan->slot_expert, plan->slot_replica, plan->expert_nrep,
                 plan->expert_rep_weight, n_src >= 2 ? plan->src_rep_weight : nullptr};
}

static int assign_impl(const int32_t* counts, const foremoe_plan* plan, int32_t* rep_begin, int32_t* slot_count,
                       int32_t* slot_offset, void* ws, size_t ws_bytes, int32_t* status, void* stream) {
  int rc = check_plan(plan, counts, rep_begin, slot_count, slot_offset, ws, ws_bytes);
  if (rc) return rc;
  const PlanDev P = plan_dev(plan);
  const int n_src = P.n_src;
  int32_t* rep_slot = (int32_t*)((char*)ws + kWsRepSlotOff);
  int32_t* vslot = (int32_t*)((char*)ws + kWsVSlotOff);
  if (n_src * plan->E <= 256)
    hipLaunchKernelGGL((assign_kernel<256, 256>), dim3(1), dim3(256), 0, (hipStream_t)stream, counts, P, rep_begin,
                       slot_count, slot_offset, vslot, rep_slot, status);
  else
    hipLaunchKernelGGL((assign_kernel<1024, FOREMOE_MAX_EXPERTS>), dim3(1), dim3(1024), 0, (hipStream_t)stream, counts,
                       P, rep_begin, slot_count, slot_offset, vslot, rep_slot, status);
  return check_launch("foremoe_assign_replicas");
}

int foremoe_assign_replicas(const int32_t* counts, const foremoe_plan* plan, int32_t* rep_begin, int32_t* slot_count,
                            int32_t* slot_offset, void* ws, size_t ws_bytes, void* stream) {
  return assign_impl(counts, plan, rep_begin, slot_count, slot_offset, ws, ws_bytes, (int32_t*)ws, stream);
}

static int histogram_assign_impl(const int32_t* ids, int64_t T, int32_t K, const foremoe_plan* plan,
                                 int32_t* counts, int32_t* rep_begin, int32_t* slot_count, int32_t* slot_offset,
                                 void* ws, size_t ws_bytes, int32_t* status, void* stream) {
  int rc = check_plan(plan, counts, rep_begin, slot_count, slot_offset, ws, ws_bytes);
  if (rc) return rc;
  const PlanDev P = plan_dev(plan);
  const int nkeys = P.n_src * P.E;
  const KeyMap km{P.E, P.n_src, K, P.n_src >= 2 ? plan->src_token_begin : nullptr};
  if (nkeys > 256) {  // large key sets: the three separate launches
    rc = histogram_common("foremoe_histogram_assign", ids, T, K, nkeys, km, counts, ws, ws_bytes, status, stream);
    if (rc) return rc;
    return assign_impl(counts, plan, rep_begin, slot_count, slot_offset, ws, ws_bytes, status, stream);
  }
  rc = check_hist("foremoe_histogram_assign", ids, T, K, nkeys, counts, ws, ws_bytes);
  if (rc) return rc;
  hipStream_t st = (hipStream_t)stream;
  const int64_t npairs = T * (int64_t)K;
  const int64_t nb = hist_blocks(npairs);
  int32_t* partial = (int32_t*)((char*)ws + kWsPartialOff);
  uint16_t* rank = (uint16_t*)((char*)ws + ws_rank_off(T, K, nkeys));
  uint32_t* ticket = (uint32_t*)ws + kWsTicketWord;
  hipLaunchKernelGGL(hist_count_kernel, dim3((unsigned)nb), dim3(kHistThreads), 0, st, ids, npairs, km, nkeys,
                     key_bits(nkeys), partial, rank, ticket);
  hipLaunchKernelGGL(hist_scan_assign_kernel, dim3(nkeys + 1), dim3(kHistThreads), 0, st, partial, nb, nkeys, counts,
                     ticket, P, rep_begin, slot_count, slot_offset,
                     (int32_t*)((char*)ws + kWsVSlotOff), (int32_t*)((char*)ws + kWsRepSlotOff), status);
  return check_launch("foremoe_histogram_assign");
}

int foremoe_histogram_assign(const int32_t* ids, int64_t T, int32_t K, const foremoe_plan* plan, int32_t* counts,
                             int32_t* rep_begin, int32_t* slot_count, int32_t* slot_offset, void* ws, size_t ws_bytes,
                             void* stream) {
  return histogram_assign_impl(ids, T, K, plan, counts, rep_begin, slot_count, slot_offset, ws, ws_bytes,
                               (int32_t*)ws, stream);
}

static int check_permute(const void* x, foremoe_dtype dtype, int64_t T, int32_t d, const int32_t* ids, int32_t K,
                         const foremoe_plan* plan, const int32_t* rep_begin, const int32_t* slot_offset,
                         int64_t n_cap, void* x_perm, int32_t* row_to_pair, int32_t* pair_to_row, void* ws,
                         size_t ws_bytes) {
  REQUIRE(plan, "permute: plan is NULL");
  REQUIRE(dtype == FOREMOE_F32 || dtype == FOREMOE_BF16, "permute: bad dtype");
  REQUIRE(T >= 0 && n_cap >= 0 && d >= 1, "permute: bad sizes");
  REQUIRE(K >= 1 && K <= FOREMOE_MAX_TOPK, "permute: K out of range");
  REQUIRE(T * (int64_t)K < (int64_t)INT_MAX && n_cap < (int64_t)INT_MAX, "permute: sizes must be below 2^31");
  REQUIRE(plan->E >= 1 && plan->E <= FOREMOE_MAX_EXPERTS, "permute: E out of range");
  REQUIRE(plan->S >= 0 && plan->S <= FOREMOE_MAX_SLOTS, "permute: S out of range");
  REQUIRE(plan->R_max >= 1 && plan->R_max <= FOREMOE_MAX_REPLICAS, "permute: R_max out of range");
  REQUIRE(rep_begin && slot_offset && ws, "permute: NULL buffer");
  REQUIRE(T == 0 || (x && ids && pair_to_row), "permute: NULL input");
  REQUIRE(n_cap == 0 || (x_perm && row_to_pair), "permute: NULL output");
  const int esz = dtype == FOREMOE_BF16 ? 2 : 4;
  if ((int64_t)d * esz % 16 != 0)
    return set_error(FOREMOE_EUNSUPPORTED, "permute: row of %d elements is not a multiple of 16 bytes", d);
  const int n_src = plan->n_src < 1 ? 1 : plan->n_src;
  if (n_src >= 2) {
    REQUIRE(n_src <= FOREMOE_MAX_SOURCES && (int64_t)n_src * plan->E <= FOREMOE_MAX_EXPERTS &&
                (int64_t)n_src * plan->S <= FOREMOE_MAX_SLOTS,
            "permute: n_src out of range");
    REQUIRE(plan->src_token_begin, "permute: plan->src_token_begin is NULL");
  }
  REQUIRE(ws_bytes >= ws_bytes_needed(T, K, n_src * plan->E), "permute: workspace too small");
  return FOREMOE_OK;
}

static int permute_impl(const void* x, foremoe_dtype dtype, int64_t T, int32_t d, const int32_t* ids, int32_t K,
                        const foremoe_plan* plan, const int32_t* rep_begin, const int32_t* slot_offset, int64_t n_cap,
                        void* x_perm, int32_t* row_to_pair, int32_t* pair_to_row, void* ws, size_t ws_bytes,
                        int32_t* status, void* stream) {
  int rc = check_permute(x, dtype, T, d, ids, K, plan, rep_begin, slot_offset, n_cap, x_perm, row_to_pair,
                         pair_to_row, ws, ws_bytes);
  if (rc) return rc;
  const int esz = dtype == FOREMOE_BF16 ? 2 : 4;
  const int n_src = plan->n_src < 1 ? 1 : plan->n_src;
  const int nkeys = n_src * plan->E;
  hipStream_t st = (hipStream_t)stream;
  const int64_t npairs = T * (int64_t)K;
  const int32_t* rep_slot = (const int32_t*)((char*)ws + kWsRepSlotOff);
  const int32_t* base = (const int32_t*)((char*)ws + kWsPartialOff);
  const uint16_t* rank = (const uint16_t*)((char*)ws + ws_rank_off(T, K, nkeys));
  // rows come from the virtual slots' offsets (the slot offsets themselves
  // with one source)
  const int32_t* row_off = n_src >= 2 ? (const int32_t*)((char*)ws + kWsVSlotOff) : slot_offset;
  const KeyMap km{plan->E, n_src, K, n_src >= 2 ? plan->src_token_begin : nullptr};
  const int64_t vpr = (int64_t)d * esz / 16;
  const int64_t groups = (npairs + 63) / 64;
  // wavefronts per group of 64 pairs: enough to give the chip 16 per CU
  // when there are fewer groups, at most 16 (measured on the benchmark's
  // shares, 8 / 16 / 32 per CU: Qwen3 EP=8 permute 28.0 / 26.6 / 27.9 us,
  // Mixtral-8x7B 28.2 / 28.1 / 28.1 us, from 89 us with one wavefront per
  // group, DeepSeek-V3 EP=32 87 / 87 / 85 us)
  const int64_t want = (int64_t)num_cus() * 16;
  int nsub = 1;
  if (groups > 0 && groups < want) nsub = (int)((want + groups - 1) / groups);  // no pairs: one, idle
  nsub = nsub > 16 ? 16 : nsub;
  // copy passes per row: one wavefront each (at most 8)
  int ncol = (int)((vpr + 64 * kVecPerLane - 1) / (64 * kVecPerLane));
  ncol = ncol < 1 ? 1 : (ncol > 8 ? 8 : ncol);
  hipLaunchKernelGGL(permute_gather_kernel, dim3(gather_grid(groups * nsub * ncol)), dim3(256), 0, st,
                     (const uint4*)x, vpr, ids, npairs, km, nkeys, plan->R_max, base, rank, rep_begin, rep_slot,
                     row_off, n_src * plan->S, slot_offset + plan->S, n_cap, pair_to_row, row_to_pair,
                     (uint4*)x_perm, status, nsub, ncol);
  return check_launch("foremoe_permute");
}

int foremoe_permute(const void* x, foremoe_dtype dtype, int64_t T, int32_t d, const int32_t* ids, int32_t K,
                    const foremoe_plan* plan, const int32_t* rep_begin, const int32_t* slot_offset, int64_t n_cap,
                    void* x_perm, int32_t* row_to_pair, int32_t* pair_to_row, void* ws, size_t ws_bytes,
                    void* stream) {
  return permute_impl(x, dtype, T, d, ids, K, plan, rep_begin, slot_offset, n_cap, x_perm, row_to_pair, pair_to_row,
                      ws, ws_bytes, (int32_t*)ws, stream);
}

static int launch_combine(const void* y_perm, foremoe_dtype in_dtype, const int32_t* pair_to_row, const float* gates,
                          int64_t T, int32_t K, int32_t d, int64_t n_cap, void* y, foremoe_dtype out_dtype,
                          hipStream_t st) {
  const dim3 grid(gather_grid(T)), block(256);
  if (in_dtype == FOREMOE_BF16 && out_dtype == FOREMOE_BF16)
    hipLaunchKernelGGL((combine_kernel<uint16_t, uint16_t>), grid, block, 0, st, (const uint16_t*)y_perm, pair_to_row,
                       gates, T, K, d, n_cap, (uint16_t*)y);
  else if (in_dtype == FOREMOE_BF16 && out_dtype == FOREMOE_F32)
    hipLaunchKernelGGL((combine_kernel<uint16_t, float>), grid, block, 0, st, (const uint16_t*)y_perm, pair_to_row,
                       gates, T, K, d, n_cap, (float*)y);
  else if (in_dtype == FOREMOE_F32 && out_dtype == FOREMOE_F32)
    hipLaunchKernelGGL((combine_kernel<float, float>), grid, block, 0, st, (const float*)y_perm, pair_to_row, gates,
                       T, K, d, n_cap, (float*)y);
  else
    return set_error(FOREMOE_EUNSUPPORTED, "combine: fp32 input with bf16 output is not supported");
  return FOREMOE_OK;
}

static int check_gather_args(const char* who, foremoe_dtype in_dtype, foremoe_dtype out_dtype, int64_t T, int32_t K,
                             int32_t d, int64_t n_cap) {
  REQUIRE(in_dtype == FOREMOE_F32 || in_dtype == FOREMOE_BF16, "%s: bad input dtype", who);
  REQUIRE(out_dtype == FOREMOE_F32 || out_dtype == FOREMOE_BF16, "%s: bad output dtype", who);
  REQUIRE(T >= 0 && d >= 1 && n_cap >= 0, "%s: bad sizes", who);
  REQUIRE(K >= 1 && K <= FOREMOE_MAX_TOPK, "%s: K out of range", who);
  REQUIRE(T * (int64_t)K < (int64_t)INT_MAX && n_cap < (int64_t)INT_MAX, "%s: sizes must be below 2^31", who);
  const int ve = in_dtype == FOREMOE_BF16 ? 8 : 4;
  if (d % ve != 0) return set_error(FOREMOE_EUNSUPPORTED, "%s: d=%d must be a multiple of %d", who, d, ve);
  return FOREMOE_OK;
}

int foremoe_combine(const void* y_perm, foremoe_dtype in_dtype, const int32_t* pair_to_row, const float* gates,
                    int64_t T, int32_t K, int32_t d, int64_t n_cap, void* y, foremoe_dtype out_dtype, void* stream) {
  int rc = check_gather_args("combine", in_dtype, out_dtype, T, K, d, n_cap);
  if (rc) return rc;
  REQUIRE(T == 0 || (pair_to_row && gates && y), "combine: NULL buffer");
  REQUIRE(T == 0 || n_cap == 0 || y_perm, "combine: y_perm is NULL");
  if (T == 0) return FOREMOE_OK;
  rc = launch_combine(y_perm, in_dtype, pair_to_row, gates, T, K, d, n_cap, y, out_dtype, (hipStream_t)stream);
  if (rc) return rc;
  return check_launch("foremoe_combine");
}

int foremoe_permute_bwd(const void* dx_perm, foremoe_dtype in_dtype, const int32_t* pair_to_row, int64_t T, int32_t K,
                        int32_t d, int64_t n_cap, void* dx, foremoe_dtype out_dtype, void* stream) {
  int rc = check_gather_args("permute_bwd", in_dtype, out_dtype, T, K, d, n_cap);
  if (rc) return rc;
  REQUIRE(T == 0 || (pair_to_row && dx), "permute_bwd: NULL buffer");
  REQUIRE(T == 0 || n_cap == 0 || dx_perm, "permute_bwd: dx_perm is NULL");
  if (T == 0) return FOREMOE_OK;
  rc = launch_combine(dx_perm, in_dtype, pair_to_row, nullptr, T, K, d, n_cap, dx, out_dtype, (hipStream_t)stream);
  if (rc) return rc;
  return check_launch("foremoe_permute_bwd");
}

int foremoe_combine_bwd(const void* dy, const void* y_perm, foremoe_dtype dtype, const int32_t* pair_to_row,
                        const float* gates, int64_t T, int32_t K, int32_t d, int64_t n_cap, void* dy_perm,
                        float* dgates, void* stream) {
  int rc = check_gather_args("combine_bwd", dtype, dtype, T, K, d, n_cap);
  if (rc) return rc;
  REQUIRE(T == 0 || (dy && pair_to_row && gates), "combine_bwd: NULL input");
  REQUIRE(T == 0 || n_cap == 0 || dy_perm, "combine_bwd: dy_perm is NULL");
  REQUIRE(!dgates || T == 0 || n_cap == 0 || y_perm, "combine_bwd: dgates needs y_perm");
  if (T == 0) return FOREMOE_OK;
  hipStream_t st = (hipStream_t)stream;
  const dim3 grid(gather_grid(T)), block(256);
  if (dtype == FOREMOE_BF16)
    hipLaunchKernelGGL(combine_bwd_kernel<uint16_t>, grid, block, 0, st, (const uint16_t*)dy, (const uint16_t*)y_perm,
                       pair_to_row, gates, T, K, d, n_cap, (uint16_t*)dy_perm, dgates);
  else
    hipLaunchKernelGGL(combine_bwd_kernel<float>, grid, block, 0, st, (const float*)dy, (const float*)y_perm,
                       pair_to_row, gates, T, K, d, n_cap, (float*)dy_perm, dgates);
  return check_launch("foremoe_combine_bwd");
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Steps 1-3 without a caller workspace: the workspace of foremoe_histogram_assign
// and foremoe_permute lives in a file-scope device array instead, for callers
// that cannot allocate device memory.
// ---------------------------------------------------------------------------
namespace foremoe {
namespace {
constexpr size_t kStaticScratchBytes = (size_t)8 << 20;  // FOREMOE_STATIC_SCRATCH_BYTES
constexpr int kMaxStaticDevices = 64;
static_assert(kStaticScratchBytes == FOREMOE_STATIC_SCRATCH_BYTES, "header and library disagree");
}  // namespace
}  // namespace foremoe

// Every device the library runs on holds its own copy of this array until the
// process ends. In host code `scratch` names a host-side stand-in, never the
// device memory: kernels receive the per-device address from
// hipGetSymbolAddress below.
static __device__ __align__(256) unsigned char scratch[foremoe::kStaticScratchBytes];

static std::mutex g_scratch_mu;
static void* g_scratch_ptr[foremoe::kMaxStaticDevices];

// The current device's address of `scratch`, looked up once per device with
// that device current.
static int static_scratch_ptr(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return set_error(FOREMOE_EHIP, "dispatch_static: hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= foremoe::kMaxStaticDevices)
    return set_error(FOREMOE_EUNSUPPORTED, "dispatch_static: device %d above %d", dev, foremoe::kMaxStaticDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return set_error(FOREMOE_EHIP, "dispatch_static: hipGetSymbolAddress: %s", hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return FOREMOE_OK;
}

extern "C" {

int foremoe_dispatch_static(const int32_t* ids, int64_t T, int32_t K, const foremoe_plan* plan, const void* x,
                            foremoe_dtype dtype, int32_t d, int64_t n_cap, int32_t* counts, int32_t* rep_begin,
                            int32_t* slot_count, int32_t* slot_offset, void* x_perm, int32_t* row_to_pair,
                            int32_t* pair_to_row, int32_t* status, void* stream) {
  REQUIRE(plan, "dispatch_static: plan is NULL");
  REQUIRE(T >= 0 && K >= 1 && K <= FOREMOE_MAX_TOPK, "dispatch_static: T or K out of range");
  REQUIRE(T * (int64_t)K < (int64_t)INT_MAX, "dispatch_static: T*K must be below 2^31");
  REQUIRE(plan->E >= 1 && plan->E <= FOREMOE_MAX_EXPERTS, "dispatch_static: E=%d out of range", plan->E);
  const int n_src = plan->n_src < 1 ? 1 : plan->n_src;
  REQUIRE(n_src <= FOREMOE_MAX_SOURCES && (int64_t)n_src * plan->E <= FOREMOE_MAX_EXPERTS,
          "dispatch_static: n_src * E above %d", FOREMOE_MAX_EXPERTS);
  const size_t need = ws_bytes_needed(T, K, n_src * plan->E);
  REQUIRE(need <= kStaticScratchBytes,
          "dispatch_static: %lld pairs over %d keys need %zu bytes of scratch, above the %zu of the static array",
          (long long)(T * K), n_src * plan->E, need, kStaticScratchBytes);
  void* ws = nullptr;
  int rc = static_scratch_ptr(&ws);
  if (rc) return rc;
  // every argument of both steps is checked before anything is launched
  rc = check_plan(plan, counts, rep_begin, slot_count, slot_offset, ws, kStaticScratchBytes);
  if (rc) return rc;
  rc = check_hist("dispatch_static", ids, T, K, n_src * plan->E, counts, ws, kStaticScratchBytes);
  if (rc) return rc;
  rc = check_permute(x, dtype, T, d, ids, K, plan, rep_begin, slot_offset, n_cap, x_perm, row_to_pair, pair_to_row,
                     ws, kStaticScratchBytes);
  if (rc) return rc;
  // status words into the caller's array, else into the scratch header
  int32_t* st = status ? status : (int32_t*)ws;
  rc = histogram_assign_impl(ids, T, K, plan, counts, rep_begin, slot_count, slot_offset, ws, kStaticScratchBytes, st,
                             stream);
  if (rc) return rc;
  return permute_impl(x, dtype, T, d, ids, K, plan, rep_begin, slot_offset, n_cap, x_perm, row_to_pair, pair_to_row,
                      ws, kStaticScratchBytes, st, stream);
}

}  // extern "C"
