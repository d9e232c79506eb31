/*
 * foremoe.h - C ABI of the per-micro-step MoE expert layer on one MI355X.
 *
 * ForeMoE (arXiv 2606.11867) balances MoE load per micro-step by placing
 * experts and expert replicas in "slots" (Sec. 7, Terminology) according to
 * the routing recorded during rollout (Sec. 5, Routing Collector). This
 * library runs what one GPU does with such a placement, in five steps:
 *
 *   1. foremoe_histogram        tokens per expert from the recorded top-K ids
 *   2. foremoe_assign_replicas  contiguous split of each expert's token list
 *                               over its replicas (token assignment r_{s,e,j},
 *                               Sec. 7.2 and Sec. 8 Stage 4)
 *   3. foremoe_permute          gather tokens into slot-contiguous order
 *   4. foremoe_grouped_ffn_*    SwiGLU expert FFN over the local slots
 *                               (App. A): forward, dgrad and wgrad; replica
 *                               weight gradients are summed into the main
 *                               expert (Sec. 6.2, Copy-in)
 *   5. foremoe_combine          gate-weighted sum back to token order (Sec. 2.1)
 *   plus foremoe_combine_bwd / foremoe_permute_bwd for the policy-update
 *   backward (Sec. 7.1: the backward repeats dispatch and combine).
 *
 * Conventions (all entry points):
 *  - Every pointer argument is a DEVICE pointer unless stated otherwise; the
 *    caller owns every buffer. The library never allocates device memory and
 *    keeps no state besides a per-thread error message and the cached
 *    compute-unit count of each device; no call changes what a later call
 *    does.
 *  - Every call is asynchronous on `stream` (a hipStream_t; NULL = the null
 *    stream) and never synchronises the host. Sizes that depend on the
 *    routing (N = local pairs, slot offsets) stay on the device.
 *  - Return value: FOREMOE_OK, or a negative status. Arguments are checked
 *    on the host before any launch; on error nothing is launched and
 *    foremoe_last_error() describes the problem. No exception crosses the ABI.
 *  - Layouts are row-major. Index types are int32. "bf16" is bfloat16.
 *  - Results are deterministic: no floating-point atomics are used, so two
 *    calls with the same inputs give bitwise identical outputs.
 *  - Thread-safe; calls on the same buffers must be ordered by the caller.
 */
#ifndef FOREMOE_H
#define FOREMOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define FOREMOE_OK 0
#define FOREMOE_EINVAL (-1)       /* bad argument (null pointer, bad size)          */
#define FOREMOE_EUNSUPPORTED (-2) /* valid but unsupported shape or dtype            */
#define FOREMOE_EHIP (-3)         /* a HIP launch failed                             */

/* Limits checked on the host. */
#define FOREMOE_MAX_EXPERTS 1024
#define FOREMOE_MAX_SLOTS 1024
#define FOREMOE_MAX_REPLICAS 16
#define FOREMOE_MAX_TOPK 64
#define FOREMOE_MAX_SOURCES 64
#define FOREMOE_MAX_WGRAD_STEPS 16

typedef enum foremoe_dtype {
  FOREMOE_F32 = 0,
  FOREMOE_BF16 = 1
} foremoe_dtype;

/*
 * One micro-step's placement on this GPU (Sec. 7, Terminology; Table 1:
 * x_{e,j} and r_{s,e,j}). A host struct whose arrays are DEVICE arrays.
 *
 *  E                  experts in the model, 1..FOREMOE_MAX_EXPERTS
 *  S                  local slots, 0..FOREMOE_MAX_SLOTS
 *  R_max              row length of expert_rep_weight, 1..FOREMOE_MAX_REPLICAS
 *  slot_expert[S]     expert held by slot j
 *  slot_replica[S]    which replica of that expert slot j holds (0-based)
 *  expert_nrep[E]     replicas R_e of expert e in the whole EP group, local
 *                     or not (1..R_max)
 *  expert_rep_weight  [E * R_max] integer split weights (>= 0, positive sum
 *                     over the first R_e entries), or NULL for equal split
 *  slot_widx[S]       weight index (0..W-1) slot j computes with; a replica
 *                     may alias its source expert's weights
 *  slot_gidx[S]       gradient index (0..G-1) slot j accumulates into: the
 *                     main expert of slot j's expert (Sec. 6.2)
 *  n_src              source ranks of the per-source split (0 or 1: one
 *                     source, the arrays below unused), 2..FOREMOE_MAX_SOURCES
 *                     with n_src * E <= FOREMOE_MAX_EXPERTS and
 *                     n_src * S <= FOREMOE_MAX_SLOTS
 *  src_token_begin    [n_src + 1] first token of each source rank (Sec. 7.2:
 *                     r_{s,e,j} is set per source rank s): source s owns the
 *                     tokens [src_token_begin[s], src_token_begin[s+1]),
 *                     nondecreasing from 0 to T (pairs of tokens outside it
 *                     count as invalid ids)
 *  src_rep_weight     [n_src * E * R_max] integer split weights per (source,
 *                     expert), e.g. a planner's water-filled token counts
 *                     (App. D Stage 4), or NULL: expert_rep_weight for every
 *                     source. All-zero weights are an error only when the
 *                     (source, expert) block has pairs.
 *
 * Errors in the device arrays (a slot naming an expert or replica out of
 * range, two slots holding the same replica, a zero weight sum) cannot be
 * seen by the host check; the device counts them in the workspace status
 * word FOREMOE_WS_PLAN_ERRORS and treats the entry as absent/equal-split.
 */
typedef struct foremoe_plan {
  int32_t E;
  int32_t S;
  int32_t R_max;
  int32_t n_src;
  const int32_t* slot_expert;
  const int32_t* slot_replica;
  const int32_t* expert_nrep;
  const int32_t* expert_rep_weight;
  const int32_t* slot_widx;
  const int32_t* slot_gidx;
  const int32_t* src_token_begin;
  const int32_t* src_rep_weight;
} foremoe_plan;

/*
 * Workspace. foremoe_histogram, foremoe_assign_replicas and foremoe_permute
 * of one micro-step share one caller-owned device workspace of at least
 * foremoe_workspace_size(T, K, E) bytes (256-byte aligned; returns 0 for
 * invalid sizes; for a per-source plan pass n_src * E as E). Its first 256
 * bytes are int32 status words (read them after the stream completes):
 */
#define FOREMOE_WS_INVALID_IDS 0  /* ids outside [-1, E): skipped, written by histogram */
#define FOREMOE_WS_DROPPED 1      /* local pairs beyond n_cap, written by permute       */
#define FOREMOE_WS_PLAN_ERRORS 2  /* device-side plan errors, written by assign         */
/* Word 63 is the arrival ticket of foremoe_histogram_assign; that call's
 * first kernel zeroes it, so a workspace needs no initialisation and a stale
 * ticket (a workspace not zero-filled, an earlier call that did not
 * complete) cannot misfire. */
size_t foremoe_workspace_size(int64_t T, int32_t K, int32_t E);

/*
 * Step 1 (Sec. 5 Routing Collector; load w_e of Table 1).
 * ids     [T, K] int32, row-major, pair p = t*K + k. -1 = padding (skipped);
 *         any other id outside [0, E) is invalid: skipped and counted in
 *         FOREMOE_WS_INVALID_IDS.
 * counts  [E] int32 out: counts[e] = #pairs with ids[p] == e over all T tokens.
 * Also fills the workspace with per-block partial counts and every pair's
 * rank within its block, both used by permute.
 * T >= 0, 1 <= K <= FOREMOE_MAX_TOPK, T*K < 2^31.
 */
int foremoe_histogram(const int32_t* ids, int64_t T, int32_t K, int32_t E,
                      int32_t* counts, void* ws, size_t ws_bytes, void* stream);

/*
 * Step 1 per source rank (Sec. 7.2, load w_{s,e} of Table 1), for plans with
 * n_src >= 2: counts [n_src, E] int32 out, counts[s][e] = #pairs of the
 * tokens [src_token_begin[s], src_token_begin[s+1]) with ids[p] == e.
 * src_token_begin [n_src + 1] device array as in foremoe_plan. Fills the
 * workspace (sized for n_src * E experts) for foremoe_permute of such a plan.
 */
int foremoe_histogram_src(const int32_t* ids, int64_t T, int32_t K, int32_t E, int32_t n_src,
                          const int32_t* src_token_begin, int32_t* counts, void* ws,
                          size_t ws_bytes, void* stream);

/*
 * Step 2 (Sec. 7.2 token conservation; Sec. 8 Stage 4; App. D Stage 4).
 * For expert e with R_e replicas and weights w (equal if NULL), replica r
 * takes the contiguous block [B_r, B_{r+1}) of e's token list (ascending
 * pair index), B_r = floor(n_e * (w_0 + .. + w_{r-1}) / (w_0 + .. + w_{R_e-1})).
 * rep_begin   [E, R_max+1] int32 out: B_0..B_{R_e}, then n_e up to R_max.
 * slot_count  [S] int32 out: tokens of slot j = B_{r+1} - B_r of its replica.
 * slot_offset [S+1] int32 out: exclusive prefix sum of slot_count in slot
 *             order; slot_offset[S] = N, the local pairs of this GPU.
 * ws          the workspace foremoe_histogram filled for the same ids.
 * Per-source plan (n_src >= 2): counts is [n_src, E] from
 * foremoe_histogram_src, the split is done for every (source, expert) block
 * with that source's weights, rep_begin is [n_src, E, R_max+1], and a slot
 * takes its replica's blocks source by source (so its rows stay in
 * ascending pair order); slot_count sums the blocks.
 */
int foremoe_assign_replicas(const int32_t* counts, const foremoe_plan* plan,
                            int32_t* rep_begin, int32_t* slot_count, int32_t* slot_offset,
                            void* ws, size_t ws_bytes, void* stream);

/*
 * Steps 1 and 2 in one call (Sec. 5 Routing Collector counts; Sec. 7.2
 * replica split): the same outputs as foremoe_histogram (plan->n_src < 2)
 * or foremoe_histogram_src (plan->n_src >= 2, sources from
 * plan->src_token_begin) into counts [n_src * E], followed by
 * foremoe_assign_replicas with the same plan, workspace and stream. With up
 * to 256 keys this is two launches instead of three: the per-key column
 * scan and the replica split share one, where the last workgroup to finish
 * the scan does the split (a ticket in workspace status word 63, see
 * above). Larger key sets run the three launches. Same argument rules and
 * errors as the two calls it replaces.
 */
int foremoe_histogram_assign(const int32_t* ids, int64_t T, int32_t K, const foremoe_plan* plan,
                             int32_t* counts, int32_t* rep_begin, int32_t* slot_count,
                             int32_t* slot_offset, void* ws, size_t ws_bytes, void* stream);

/*
 * Step 3 (Sec. 9, replica-aware token dispatch; one GPU's half of it).
 * Pair p with expert e is the q-th entry of e's token list and belongs to
 * replica r with B_r <= q < B_{r+1}. If slot j holds (e, r) here, its row is
 * row = slot_offset[j] + q - B_r and
 *   x_perm[row, :] = x[p / K, :]   (bitwise copy)
 *   row_to_pair[row] = p,  pair_to_row[p] = row;
 * otherwise pair_to_row[p] = -1. Rows >= N are not written. Pairs whose row
 * would be >= n_cap are dropped (pair_to_row = -1) and counted in
 * FOREMOE_WS_DROPPED.
 * x        [T, d] of `dtype`; d % 8 == 0 (bf16) or d % 4 == 0 (f32).
 * x_perm   [n_cap, d] of `dtype`; row_to_pair [n_cap]; pair_to_row [T*K].
 * ws       the workspace filled by foremoe_histogram and
 *          foremoe_assign_replicas for the same ids and plan.
 * Per-source plan: q is the rank within the pair's (source, expert) list,
 * B the bounds of that block, and the row follows the source's earlier
 * blocks in slot j (foremoe_histogram_src must have filled ws).
 */
int foremoe_permute(const void* x, foremoe_dtype dtype, int64_t T, int32_t d,
                    const int32_t* ids, int32_t K, const foremoe_plan* plan,
                    const int32_t* rep_begin, const int32_t* slot_offset, int64_t n_cap,
                    void* x_perm, int32_t* row_to_pair, int32_t* pair_to_row,
                    void* ws, size_t ws_bytes, void* stream);

/*
 * Steps 1-3 without a workspace argument, for callers that cannot allocate
 * device memory (code under stream capture, serving loops that forbid
 * allocation): the same work and outputs as foremoe_histogram_assign
 * followed by foremoe_permute with the same arguments, bitwise, and the same
 * argument rules and errors. The workspace of those two calls lives in a
 * device array of FOREMOE_STATIC_SCRATCH_BYTES that the library holds on
 * every device it runs on until the process ends; the call allocates
 * nothing. Inputs whose workspace would exceed it, i.e.
 * foremoe_workspace_size(T, K, n_src * E) > FOREMOE_STATIC_SCRATCH_BYTES
 * (about 2.7 M pairs at E = 128, 0.83 M pairs at 1024 keys), are rejected with
 * FOREMOE_EINVAL before anything is launched.
 * status  int32 [3] out or NULL: the status words FOREMOE_WS_INVALID_IDS,
 *         FOREMOE_WS_DROPPED and FOREMOE_WS_PLAN_ERRORS of the call.
 * Every call on one device shares that device's array, which keeps the last
 * call's contents: calls that overlap in time on one device (two streams,
 * two host threads) race and give wrong results; order them.
 */
#define FOREMOE_STATIC_SCRATCH_BYTES ((size_t)8 << 20)
int foremoe_dispatch_static(const int32_t* ids, int64_t T, int32_t K, const foremoe_plan* plan,
                            const void* x, foremoe_dtype dtype, int32_t d, int64_t n_cap,
                            int32_t* counts, int32_t* rep_begin, int32_t* slot_count,
                            int32_t* slot_offset, void* x_perm, int32_t* row_to_pair,
                            int32_t* pair_to_row, int32_t* status, void* stream);

/*
 * Step 4, forward (App. A: SwiGLU expert with gate, up and down matrices).
 * For each slot j, rows [slot_offset[j], slot_offset[j+1]) (clamped to
 * n_cap), with w = slot_widx[j] (a slot with w outside [0, W) is skipped by
 * this and the input-gradient calls: its rows of every output keep what
 * they held):
 *   A = X Wg[w]^T, U = X Wu[w]^T      (fp32 accumulate)
 *   H = silu(A) * U,  silu(a) = a / (1 + exp(-a))
 *   Y = H Wd[w]^T
 * x_perm     [n_cap, d]
 * w_gate_up  [W, 2F, d]: rows [0, F) are Wg[w], rows [F, 2F) are Wu[w]
 * w_down     [W, d, F]
 * h          [n_cap, F] out (kept for the weight gradient)
 * y_perm     [n_cap, d] out
 * save_au    [n_cap, 2F] out or NULL: A in columns [0, F), U in [F, 2F)
 *            (needed by foremoe_grouped_ffn_dgrad)
 * All tensors are `dtype`. bf16 runs on bf16 MFMA with fp32 accumulation
 * and needs d % 128 == 0, F % 128 == 0 and (n_cap + 256) * max(d, 2F) * 2
 * below 2^32 (else FOREMOE_EUNSUPPORTED); f32 accepts any d, F >= 1.
 * 0 <= S <= FOREMOE_MAX_SLOTS.
 * foremoe_grouped_ffn_fwd = foremoe_ffn_gate_up_fwd then foremoe_ffn_down_fwd;
 * each of these two is a single kernel launch.
 *
 * workspace (optional, these and the input-gradient calls below): NULL, or
 * caller-owned device memory of at least foremoe_ffn_workspace_size()
 * bytes, 256-byte aligned, zero-filled before its first use (the library
 * leaves its counters at zero after every call). A last round of output
 * tiles that would occupy at most 7/16 of the GPU's CUs is cut along N into
 * half-width tiles when the tiles are 256 wide (with or without a
 * workspace). With the workspace, the (half) tiles of such a round are also
 * cut along K (in GEMMs whose K is at least 2048) into up to 4 pieces (as
 * many as keep at most 7/8 of the CUs busy), each computed by its own
 * workgroup; the last piece to finish adds the pieces' fp32 partial sums in
 * piece order and writes the tile. Results are deterministic either way and
 * equal with and without the workspace up to the fp32 summation order.
 * Calls that share a workspace
 * must not overlap in time (same stream, or ordered by events); after a
 * call that did not complete, zero the workspace again. Too small or
 * misaligned: FOREMOE_EINVAL, nothing launched. Ignored for f32.
 */
size_t foremoe_ffn_workspace_size(void);

int foremoe_grouped_ffn_fwd(const void* x_perm, foremoe_dtype dtype, int32_t d, int32_t F,
                            int32_t S, const int32_t* slot_offset, const int32_t* slot_widx,
                            int32_t W, const void* w_gate_up, const void* w_down, int64_t n_cap,
                            void* h, void* y_perm, void* save_au, void* workspace, size_t ws_bytes, void* stream);
int foremoe_ffn_gate_up_fwd(const void* x_perm, foremoe_dtype dtype, int32_t d, int32_t F,
                            int32_t S, const int32_t* slot_offset, const int32_t* slot_widx,
                            int32_t W, const void* w_gate_up, int64_t n_cap,
                            void* h, void* save_au, void* workspace, size_t ws_bytes, void* stream);
int foremoe_ffn_down_fwd(const void* h, foremoe_dtype dtype, int32_t d, int32_t F,
                         int32_t S, const int32_t* slot_offset, const int32_t* slot_widx,
                         int32_t W, const void* w_down, int64_t n_cap, void* y_perm, void* workspace, size_t ws_bytes, void* stream);

/*
 * Step 4, input gradient (chain rule of the forward above):
 *   dH = dY Wd[w];  dA = dH * U * silu'(A);  dU = dH * silu(A)
 *   dX = dA Wg[w] + dU Wu[w]
 * with silu'(a) = s + a s (1 - s), s = 1 / (1 + exp(-a)).
 * dy_perm [n_cap, d]; save_au [n_cap, 2F] from the forward;
 * d_au    [n_cap, 2F] out: dA in columns [0, F), dU in [F, 2F);
 * dx_perm [n_cap, d] out. Same dtype, shape and workspace rules as the
 * forward.
 * = foremoe_ffn_down_dgrad then foremoe_ffn_gate_up_dgrad (one launch each).
 */
int foremoe_grouped_ffn_dgrad(const void* dy_perm, const void* save_au, foremoe_dtype dtype,
                              int32_t d, int32_t F, int32_t S, const int32_t* slot_offset,
                              const int32_t* slot_widx, int32_t W, const void* w_gate_up,
                              const void* w_down, int64_t n_cap, void* d_au, void* dx_perm,
                              void* workspace, size_t ws_bytes, void* stream);
int foremoe_ffn_down_dgrad(const void* dy_perm, const void* save_au, foremoe_dtype dtype,
                           int32_t d, int32_t F, int32_t S, const int32_t* slot_offset,
                           const int32_t* slot_widx, int32_t W, const void* w_down,
                           int64_t n_cap, void* d_au, void* workspace, size_t ws_bytes, void* stream);
int foremoe_ffn_gate_up_dgrad(const void* d_au, foremoe_dtype dtype, int32_t d, int32_t F,
                              int32_t S, const int32_t* slot_offset, const int32_t* slot_widx,
                              int32_t W, const void* w_gate_up, int64_t n_cap, void* dx_perm,
                              void* workspace, size_t ws_bytes, void* stream);

/*
 * Step 4, weight gradient with main-expert accumulation (Sec. 6.2, Copy-in:
 * the partial gradients of all replicas of an expert are summed into the
 * main expert's gradient; App. A.4: fp32 gradient accumulation):
 *   dW_gate_up[g] += [dA | dU]^T X,   dW_down[g] += dY^T H
 * summed over the rows of every slot j with slot_gidx[j] == g, in slot
 * order. ACCUMULATES (+=) into fp32 dw_gate_up [G, 2F, d] and
 * dw_down [G, d, F], so gradients add up over micro-steps.
 * ws, ws_bytes: optional device scratch, caller-owned: a 256-byte header of
 *   work counters (workgroups take the next (tile, row chunk) item when they
 *   are free), then fp32 partial tiles for splitting one expert's rows over
 *   many workgroups, summed in a fixed order by a second kernel of the same
 *   call. foremoe_wgrad_workspace_size(d, F) bytes give the full split. The
 *   header must be zero-filled before the first call; every call leaves it
 *   zero again (the rest needs no initialisation). NULL/0 runs with a fixed
 *   item order and no split (slower for skewed loads, same result). Calls
 *   sharing one ws must be ordered on one stream.
 * No float atomics: each output element's summation order is fixed, so the
 * result is deterministic. 1 <= G <= FOREMOE_MAX_SLOTS.
 * = foremoe_ffn_gate_up_wgrad then foremoe_ffn_down_wgrad (each one main
 *   kernel, plus one reduction kernel when ws is given).
 */
size_t foremoe_wgrad_workspace_size(int32_t d, int32_t F);
int foremoe_grouped_ffn_wgrad(const void* x_perm, const void* h, const void* dy_perm,
                              const void* d_au, foremoe_dtype dtype, int32_t d, int32_t F,
                              int32_t S, const int32_t* slot_offset, const int32_t* slot_gidx,
                              int32_t G, int64_t n_cap, float* dw_gate_up, float* dw_down,
                              void* ws, size_t ws_bytes, void* stream);
int foremoe_ffn_gate_up_wgrad(const void* d_au, const void* x_perm, foremoe_dtype dtype,
                              int32_t d, int32_t F, int32_t S, const int32_t* slot_offset,
                              const int32_t* slot_gidx, int32_t G, int64_t n_cap,
                              float* dw_gate_up, void* ws, size_t ws_bytes, void* stream);
int foremoe_ffn_down_wgrad(const void* dy_perm, const void* h, foremoe_dtype dtype,
                           int32_t d, int32_t F, int32_t S, const int32_t* slot_offset,
                           const int32_t* slot_gidx, int32_t G, int64_t n_cap,
                           float* dw_down, void* ws, size_t ws_bytes, void* stream);

/*
 * Step 4, weight gradient of several micro-steps in one call (the same
 * accumulation as above; App. A.4: the expert gradients are summed in fp32
 * over the micro-steps of an update step). Each micro-step m contributes
 * the rows of its own slots with its own operands and slot table:
 *   dW_gate_up[g] += sum over m, then j with slot_gidx_m[j] == g, of
 *                    d_au_m[rows of j]^T x_perm_m[rows of j]
 *   dW_down[g]    += same with dy_perm_m and h_m
 * Every group's rows are taken micro-step by micro-step in the order given,
 * each micro-step's slots in slot order; the summation order is fixed, so
 * the result is deterministic. It equals the sum of one call per micro-step
 * up to fp32 rounding: one read-modify-write of dW serves all the
 * micro-steps (a launch over 4 micro-steps moves a quarter of the fp32
 * gradient traffic of 4 launches).
 * steps: host array of n_steps records (read during the call only);
 *   a, b: gate/up: d_au [n_cap, 2F] and x_perm [n_cap, d];
 *         down: dy_perm [n_cap, d] and h [n_cap, F];
 *   slot_offset [S+1], slot_gidx [S]: that micro-step's device slot table;
 *   S, n_cap: its slots and buffer rows (S == 0 or n_cap == 0: skipped).
 * part, parts (0 <= part < parts <= FOREMOE_MAX_WGRAD_STEPS): the call
 *   updates only part `part` of every dW[g]: with 256 x 256 output tiles
 *   (128 x 128 when a dimension is not a multiple of 256) numbered row-major,
 *   the tiles t with t % parts == part (the fp32 path: rows m with
 *   m % parts == part). The parts 0 .. parts-1 of the same steps together
 *   give the whole update, so one group of micro-steps can be spread over
 *   several launches. parts = 1: everything.
 * 0 <= n_steps <= FOREMOE_MAX_WGRAD_STEPS; the S of all steps add up to at
 * most FOREMOE_MAX_SLOTS. Workspace, dtype, shape and G rules as above.
 */
typedef struct foremoe_wgrad_step {
  const void* a;
  const void* b;
  const int32_t* slot_offset;
  const int32_t* slot_gidx;
  int32_t S;
  int64_t n_cap;
} foremoe_wgrad_step;

int foremoe_ffn_gate_up_wgrad_steps(const foremoe_wgrad_step* steps, int32_t n_steps,
                                    foremoe_dtype dtype, int32_t d, int32_t F, int32_t G,
                                    int32_t part, int32_t parts, float* dw_gate_up, void* ws,
                                    size_t ws_bytes, void* stream);
int foremoe_ffn_down_wgrad_steps(const foremoe_wgrad_step* steps, int32_t n_steps,
                                 foremoe_dtype dtype, int32_t d, int32_t F, int32_t G,
                                 int32_t part, int32_t parts, float* dw_down, void* ws,
                                 size_t ws_bytes, void* stream);

/*
 * Step 5 (Sec. 2.1: the output is the router-probability weighted sum of
 * the selected experts' outputs):
 *   y[t, :] = sum_{k ascending, pair_to_row[tK+k] >= 0} gates[tK+k] * Y[row, :]
 * fp32 accumulation; tokens with no local pair get a zero row (y is dense,
 * this GPU's share of the sum).
 * y_perm [n_cap, d] of in_dtype; gates [T, K] fp32; y [T, d] of out_dtype.
 */
int foremoe_combine(const void* y_perm, foremoe_dtype in_dtype, const int32_t* pair_to_row,
                    const float* gates, int64_t T, int32_t K, int32_t d, int64_t n_cap,
                    void* y, foremoe_dtype out_dtype, void* stream);

/*
 * Backward of step 5. For every pair p = tK+k with row = pair_to_row[p] >= 0:
 *   dy_perm[row, :] = gates[p] * dy[t, :]
 *   dgates[p] = <dy[t, :], y_perm[row, :]>        (fp32)
 * and dgates[p] = 0 for pairs not computed here. dgates may be NULL (then
 * y_perm is not read and may be NULL). dy [T, d], y_perm and dy_perm
 * [n_cap, d], all of `dtype`.
 */
int foremoe_combine_bwd(const void* dy, const void* y_perm, foremoe_dtype dtype,
                        const int32_t* pair_to_row, const float* gates, int64_t T, int32_t K,
                        int32_t d, int64_t n_cap, void* dy_perm, float* dgates, void* stream);

/*
 * Backward of step 3: dx[t, :] = sum_{k ascending, row >= 0} dx_perm[row, :]
 * (fp32 accumulation), zero rows for tokens with no local pair.
 * dx_perm [n_cap, d] of in_dtype; dx [T, d] of out_dtype.
 */
int foremoe_permute_bwd(const void* dx_perm, foremoe_dtype in_dtype, const int32_t* pair_to_row,
                        int64_t T, int32_t K, int32_t d, int64_t n_cap, void* dx,
                        foremoe_dtype out_dtype, void* stream);

/*
 * Expert Transfer Engine, the part one GPU runs (Sec. 6).
 *
 * Records (App. A.3: one expert's state, S_e + S_g bytes). A record holds,
 * in this order and each in the weights' own row-major layout, the parts
 * `what` selects: FOREMOE_XFER_PARAMS = the gate/up parameters [2F, d] and
 * the down parameters [d, F] in the parameter dtype (S_e = 3 d F p_w bytes);
 * FOREMOE_XFER_GRADS = the fp32 gate/up gradient [2F, d] and down gradient
 * [d, F] (S_g = 12 d F bytes, App. A.4 fp32 accumulation). Record i of a
 * buffer starts at i * foremoe_xfer_record_bytes(d, F, dtype, what)
 * (0 for invalid arguments). d * F must be a multiple of 8.
 * Index lists (widx, gidx, gmode, expert) are HOST arrays of n entries,
 * n <= FOREMOE_MAX_XFER_RECORDS; they are checked on the host before any
 * launch. Expert arrays and buffers are device memory, 16-byte aligned:
 * w_gate_up [W, 2F, d], w_down [W, d, F] (parameter dtype), dw_gate_up
 * [G, 2F, d], dw_down [G, d, F] (fp32).
 */
#define FOREMOE_XFER_PARAMS 1
#define FOREMOE_XFER_GRADS 2
#define FOREMOE_XFER_ASSIGN 0 /* the gradient target takes the record           */
#define FOREMOE_XFER_ADD 1    /* the record is added into the gradient target    */
#define FOREMOE_MAX_XFER_RECORDS 64
size_t foremoe_xfer_record_bytes(int32_t d, int32_t F, foremoe_dtype dtype, int32_t what);

/*
 * Copy-out (Sec. 6.2): pack the experts leaving this GPU into the send
 * buffer, record i holding weight slot widx[i] (with PARAMS) and gradient
 * slot gidx[i] (with GRADS). buf: at least n records. One kernel launch
 * (none for n = 0); the source arrays are only read.
 */
int foremoe_copy_out(const void* w_gate_up, const void* w_down, foremoe_dtype dtype, int32_t W,
                     const float* dw_gate_up, const float* dw_down, int32_t G, int32_t d, int32_t F,
                     int32_t n, const int32_t* widx, const int32_t* gidx, int32_t what, void* buf,
                     size_t buf_bytes, void* stream);

/*
 * Copy-in (Sec. 6.2): unpack the n records of a receive buffer. With PARAMS,
 * record i's parameters go to weight slot widx[i] (< 0: skipped; two
 * records may not name one slot). With GRADS, record i's gradient goes to
 * gradient slot gidx[i] (< 0: skipped): gmode[i] = FOREMOE_XFER_ASSIGN moves
 * it there (an expert arriving with its accumulated gradient),
 * FOREMOE_XFER_ADD adds it (a replica's partial gradient accumulated into
 * the main expert, Sec. 6.2). The records naming one gradient slot are
 * applied in record order, starting from the slot's current value, every
 * sum rounded to fp32, so the result is deterministic. One kernel launch.
 */
int foremoe_copy_in(const void* buf, size_t buf_bytes, int32_t n, const int32_t* widx,
                    const int32_t* gidx, const int32_t* gmode, int32_t what, void* w_gate_up,
                    void* w_down, foremoe_dtype dtype, int32_t W, float* dw_gate_up, float* dw_down,
                    int32_t G, int32_t d, int32_t F, void* stream);

/*
 * CPU-assisted path (Sec. 6.1), host only, synchronous, no GPU work: of
 * the n experts the next micro-step needs (needed[n], distinct), those
 * already in a weight slot (resident[W]: expert of each slot, -1 empty)
 * stay there; each missing one, in the order listed, takes the lowest slot
 * whose expert is not needed. Outputs (host): slot_of[n], the weight slot
 * of each needed expert, and the n_fetch fetches (fetch_expert[i] into
 * weight slot fetch_widx[i]), exactly the needed experts not resident.
 */
int foremoe_plan_prefetch(const int32_t* resident, int32_t W, const int32_t* needed, int32_t n,
                          int32_t* slot_of, int32_t* fetch_expert, int32_t* fetch_widx,
                          int32_t* n_fetch);

/*
 * CPU-assisted prefetch (Sec. 6.1; App. A.2): copy the parameters of
 * expert[i] from the host master copy (host_gate_up [E, 2F, d], host_down
 * [E, d, F]; HOST memory, pinned with hipHostMalloc so that the copy runs
 * asynchronously on the DMA engines) into weight slot widx[i] (distinct) of
 * the device arrays, as host-to-device copies queued on `stream` (the
 * caller's auxiliary stream, so that they overlap the current layer's work
 * on the main stream). No kernel, no GPU buffer.
 */
int foremoe_prefetch_experts(const void* host_gate_up, const void* host_down, int32_t E,
                             foremoe_dtype dtype, int32_t d, int32_t F, int32_t n,
                             const int32_t* expert, const int32_t* widx, void* w_gate_up,
                             void* w_down, int32_t W, void* stream);

/*
 * Placement planner (host only: HOST arrays, no GPU work, synchronous).
 * Produces the placement that the GPU steps consume, from the routing
 * foreseen during rollout (Sec. 5). Ranks are numbered machine-major:
 * rank r sits on machine r / R; P = M * R ranks, which are also the source
 * ranks s of the load matrices (w[s, e] = tokens of source rank s routed to
 * expert e, int32, row-major [P, E]).
 *
 *  M    machines, R ranks per machine (M * R <= 4096)
 *  N_b  base slots per rank (E <= P * N_b), N_r redundant slots per rank
 *
 * Ties are broken the same way everywhere: lowest expert id, rank id or
 * copy index among equals; all arithmetic is integer, so plans are exactly
 * reproducible. Errors: FOREMOE_EINVAL with foremoe_last_error().
 */
typedef struct foremoe_machine {
  int32_t M;
  int32_t R;
  int32_t N_b;
  int32_t N_r;
} foremoe_machine;

/*
 * Stage 1 (Sec. 8 Stage 1, Alg. 1): base rank of every expert from the
 * step's aggregate load w_agg [P, E]. Experts go, in descending aggregate
 * load, to the machine with the least
 *   c_load * (ML[m] + w_e) + c_traffic * (MC[m] + Delta_{m,e})
 * (ML: load placed on m, MC: its inbound cross-machine tokens, Delta: tokens
 * of e from other machines; c_load : c_traffic is n1*K1 : n2*K2 of the time
 * model, Sec. 7.1, as integers in [0, 2^20]) that has a free base slot, then
 * by LPT onto the machine's ranks (at most N_b each).
 * base_rank [E] out.
 */
int foremoe_plan_base(const int32_t* w_agg, int32_t E, const foremoe_machine* mc, int64_t c_load,
                      int64_t c_traffic, int32_t* base_rank);

/*
 * Policy-update Stages 2-4 (App. D, Alg. 3) for one micro-step with load
 * w [P, E], per machine:
 *   Stage 2  LPT of the machine's experts over its ranks by this load;
 *   Stage 3  R * N_r times: a replica of the expert with the largest load
 *            per copy onto the rank with the least load (copies sharing
 *            their expert's load evenly) that has a free redundant slot and
 *            no copy of that expert yet; stops when no rank qualifies;
 *   Stage 4  water-filling: replicated experts in descending load, sources
 *            in ascending order, every token unit to the copy whose rank
 *            has the least accumulated load (Sec. 7.2 r_{s,e,j} x w_{s,e}).
 * base_rank [E] in (Stage 1). C_max: copies per expert the outputs hold
 * (error if a plan needs more).
 * copy_rank [E, C_max] out: rank of copy c of expert e (copy 0 = the main
 *   expert, Sec. 6.2), -1 past the last copy.
 * counts [P, E, C_max] out: tokens of source s for expert e that copy c
 *   processes (sum over c = w[s, e]).
 * rank_load [P] out (may be NULL): tokens each rank processes.
 */
int foremoe_plan_micro_step(const int32_t* w, int32_t E, const foremoe_machine* mc,
                            const int32_t* base_rank, int32_t C_max, int32_t* copy_rank,
                            int32_t* counts, int64_t* rank_load);

/*
 * One rank's slot table from a micro-step plan (the arrays of foremoe_plan,
 * on the host): main copies on `rank` first, then replica copies on it, each
 * in ascending (expert, copy). slot_widx[j] is the index of slot j's expert
 * in local_experts (order of first appearance; use it as slot_gidx too),
 * expert_nrep[e] the copies of e in the whole group. Arrays hold max_slots
 * slots and E experts; *S_out slots and *W_out local experts are written.
 */
int foremoe_plan_rank_slots(const int32_t* copy_rank, int32_t E, int32_t C_max, int32_t rank,
                            int32_t max_slots, int32_t* slot_expert, int32_t* slot_replica,
                            int32_t* slot_widx, int32_t* expert_nrep, int32_t* local_experts,
                            int32_t* S_out, int32_t* W_out);

/*
 * Timed forms of the four row-GEMM calls (a measurement aid, not an
 * operation of the method): the same arguments, work and results as
 * foremoe_ffn_gate_up_fwd, foremoe_ffn_down_fwd, foremoe_ffn_down_dgrad and
 * foremoe_ffn_gate_up_dgrad, plus two hipEvent_t handles owned by the
 * caller (created beforehand, timing enabled; either may be NULL). The
 * events are attached to the call's one kernel launch: they are set when
 * that kernel starts and when it ends, with no separate event command in
 * the stream, so hipEventElapsedTime(start, stop) is the kernel's own
 * duration. A call that launches nothing (S == 0 or n_cap == 0) records
 * both events back to back; a call that fails before launching leaves them
 * untouched. Nothing is kept after the call returns.
 */
int foremoe_ffn_gate_up_fwd_timed(const void* x_perm, foremoe_dtype dtype, int32_t d, int32_t F,
                                  int32_t S, const int32_t* slot_offset, const int32_t* slot_widx,
                                  int32_t W, const void* w_gate_up, int64_t n_cap, void* h,
                                  void* save_au, void* workspace, size_t ws_bytes, void* stream,
                                  void* start_event, void* stop_event);
int foremoe_ffn_down_fwd_timed(const void* h, foremoe_dtype dtype, int32_t d, int32_t F, int32_t S,
                               const int32_t* slot_offset, const int32_t* slot_widx, int32_t W,
                               const void* w_down, int64_t n_cap, void* y_perm, void* workspace,
                               size_t ws_bytes, void* stream, void* start_event, void* stop_event);
int foremoe_ffn_down_dgrad_timed(const void* dy_perm, const void* save_au, foremoe_dtype dtype,
                                 int32_t d, int32_t F, int32_t S, const int32_t* slot_offset,
                                 const int32_t* slot_widx, int32_t W, const void* w_down,
                                 int64_t n_cap, void* d_au, void* workspace, size_t ws_bytes,
                                 void* stream, void* start_event, void* stop_event);
int foremoe_ffn_gate_up_dgrad_timed(const void* d_au, foremoe_dtype dtype, int32_t d, int32_t F,
                                    int32_t S, const int32_t* slot_offset, const int32_t* slot_widx,
                                    int32_t W, const void* w_gate_up, int64_t n_cap, void* dx_perm,
                                    void* workspace, size_t ws_bytes, void* stream,
                                    void* start_event, void* stop_event);

/* Utilities (host only, no GPU work). */
const char* foremoe_status_string(int status);
const char* foremoe_last_error(void); /* message of this thread's last failed call */
const char* foremoe_version(void);

#ifdef __cplusplus
}
#endif
#endif /* FOREMOE_H */
