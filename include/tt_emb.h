/*
 * tt_emb.h - C ABI of the MI355X (gfx950) Tensor-Train embedding gather.
 *
 * The operator follows FlowTT (ICCAD'26).  A table of N rows and D = d1*d2*d3
 * columns is stored as three TT cores (rank profile 1, R, R, 1).  Row g is
 * split by the mixed-radix conversion of Eq. 2 (Section 3.3) into digits
 * (i1, i2, i3), with the first factor the most significant digit, and
 * rebuilt by the chained contraction of Section 3.2 (Fig. 3):
 *     C = A . B    with A = G1[i1] (d1 x R) and B = G2[i2] (R x d2 R),
 *     E = C . D    with C viewed as (d1 d2) x R and D = G3[i3] (R x d3),
 * and rows are sum-pooled per bag into V.  The backward pass (Section 3.2,
 * Eq. 1) produces dense gradients of all three cores.  Indices are grouped by
 * their (i1, i2) prefix as in Section 3.3 (sort, exact unique, mixed-radix
 * digits, run-length encoding of prefixes) so that C is built once per
 * prefix group and reused for every row of the group.
 *
 * Layouts (float32, row-major, all tables of one call contiguous):
 *     G1 [T][n1][d1][R]
 *     G2 [T][n2][R][d2][R]
 *     G3 [T][n3][R][d3]
 *     out, grad_out [T][B][D], element (t, b, j1*d2*d3 + j2*d3 + j3)
 *     indices int64 [num_indices]: the row ids of all tables, table-major
 *     offsets int64 [T*B + 1]: bag t*B+b of table t covers
 *         indices[offsets[t*B+b] .. offsets[t*B+b+1]); offsets[0] = 0 and
 *         offsets[T*B] = num_indices.  NULL offsets means one index per bag
 *         (num_indices = T*B).
 *
 * Ownership.  The caller owns every device buffer (cores, indices, offsets,
 * outputs, gradients, workspace).  The handle holds host-side metadata only;
 * creating it touches no device.  tt_emb_group, tt_emb_forward,
 * tt_emb_backward, tt_emb_backward_sgd and tt_emb_sgd enqueue kernels on
 * `stream` (a hipStream_t; NULL = the default stream) and return without
 * synchronising; they allocate and free nothing.  One handle and one workspace serve one stream at a time.
 * Device pointers to float data must be 16-byte aligned, to int64 data
 * 8-byte aligned, and the workspace 256-byte aligned.
 *
 * Errors.  Host-checkable faults (NULL pointers, bad sizes or factors,
 * workspace too small, misalignment) return a status and launch nothing.  A
 * failing HIP call returns TT_EMB_EHIP.  Faults only the device can see (an
 * index outside [0, N), offsets that are not monotone within
 * [0, num_indices]) set a sticky error word in the workspace; the offending
 * occurrence contributes nothing, and tt_emb_check_errors reports
 * TT_EMB_ERANGE.  The word is cleared when a grouping starts (tt_emb_group,
 * or forward/backward with reuse_grouping = 0) and stays set through calls
 * that reuse that grouping.  No C++ exception crosses this interface.
 */
#ifndef TT_EMB_H
#define TT_EMB_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct tt_emb_s* tt_emb_handle;

typedef enum {
  TT_EMB_OK = 0,
  TT_EMB_EINVAL = 1,      /* bad argument: NULL pointer, size, factor, alignment, small workspace */
  TT_EMB_ENOMEM = 2,      /* host allocation of the handle failed */
  TT_EMB_EHIP = 3,        /* a HIP runtime call or kernel launch failed */
  TT_EMB_ERANGE = 4,      /* device saw an index outside [0, N) or malformed offsets */
  TT_EMB_EUNSUPPORTED = 5, /* shape beyond this library's limits (see tt_emb_create) */
  TT_EMB_ESCRATCH = 6      /* call larger than the static scratch of tt_emb_forward_noalloc */
} tt_emb_status;

/* Shape of the tables served by one handle.  Every table of a call has the
 * same TT shape (tables are batched into one launch, one table per key
 * range; Section 4.1 evaluates many equally-shaped tables). */
typedef struct {
  int32_t num_tables;      /* T >= 1 */
  int64_t num_rows;        /* N, 1 <= N <= n1*n2*n3 */
  int32_t row_factors[3];  /* (n1, n2, n3) >= 1; n1 is the most significant digit (Eq. 2) */
  int32_t dim_factors[3];  /* (d1, d2, d3) >= 1; j1 is the most significant output digit */
  int32_t rank;            /* R = r1 = r2 >= 1 (r0 = r3 = 1) */
  int64_t max_indices;     /* largest num_indices of any call (all tables together) */
  int64_t max_bags;        /* largest num_bags (bags per table) of any call */
} tt_emb_desc;

/* Validate `desc` and create a handle (host memory only).
 * Limits: T * n1*n2*n3 < 2^32 - 1; T * n1 * n2 < 2^28; max_indices < 2^31;
 * T * max_bags < 2^31; R <= 64; d1*d2*R <= 8192; D <= 4096.
 * Returns TT_EMB_EINVAL for non-positive sizes or N > n1*n2*n3,
 * TT_EMB_EUNSUPPORTED beyond the limits, TT_EMB_ENOMEM on allocation failure. */
tt_emb_status tt_emb_create(const tt_emb_desc* desc, tt_emb_handle* out);

/* Release a handle.  NULL is accepted. */
tt_emb_status tt_emb_destroy(tt_emb_handle h);

/* Reuse levels of the gather, for the reuse ablation of Section 4.5:
 *   TT_EMB_REUSE_PREFIX  (default) exact dedup and prefix groups: C = A.B once
 *                        per prefix group (Section 3.3);
 *   TT_EMB_REUSE_UNIQUE  exact dedup only: C recomputed for every unique row;
 *   TT_EMB_REUSE_NONE    no dedup: every occurrence is its own row and
 *                        recomputes C.
 * All three compute the same function.  Set the level before
 * tt_emb_workspace_size (the workspace grows for the two ablation levels) and
 * before the first call that uses a workspace.  Host only; returns
 * TT_EMB_EINVAL for an unknown level. */
typedef enum { TT_EMB_REUSE_PREFIX = 0, TT_EMB_REUSE_UNIQUE = 1, TT_EMB_REUSE_NONE = 2 } tt_emb_reuse;
tt_emb_status tt_emb_set_reuse(tt_emb_handle h, int level);

/* Work distribution of the fused kernels, for the scheduling ablation of
 * Section 4.4:
 *   TT_EMB_SCHED_STEAL       (default) persistent workers take chunks of
 *                            prefix groups from shared queues and steal from
 *                            other queues when theirs runs dry (Section 3.4);
 *   TT_EMB_SCHED_STATIC      each worker takes a fixed contiguous share of
 *                            the chunks (equal counts, no work moves);
 *   TT_EMB_SCHED_STEAL_CKPT  stealing plus inter-worker reuse of the
 *                            intermediate C (Section 3.5): a worker that
 *                            builds C for a prefix group publishes it in a
 *                            small table in the workspace (a few KB per
 *                            resident worker, L2-resident), and a worker that
 *                            meets the same group later reloads it instead of
 *                            recomputing it, whenever the entry still holds
 *                            that group;
 *   TT_EMB_SCHED_GROUP       static prefix mapping, the baseline of Section
 *                            4.4: every prefix group is one work unit of its
 *                            own, never split across workers (a group of more
 *                            than 64 work slices, i.e. more than 2,048 unique
 *                            rows, is cut into 64-slice pieces), and each
 *                            worker takes a fixed contiguous share of the
 *                            groups.
 * The checkpoint applies to the kernels that keep one C per worker (the
 * generic kernels); the MFMA kernels (forward and backward for d = (4,4,8)
 * with R = 32 or 64) build C for four slices per matrix-core tile and treat
 * STEAL_CKPT as STEAL.  All
 * modes compute the same function.  Host only; may be changed between calls,
 * except that TT_EMB_SCHED_GROUP cuts the work list in the grouping and needs a
 * larger workspace: set it before tt_emb_workspace_size, and a grouping made
 * in another mode is not reused across a switch into or out of it.  Returns
 * TT_EMB_EINVAL for an unknown mode. */
typedef enum {
  TT_EMB_SCHED_STEAL = 0,
  TT_EMB_SCHED_STATIC = 1,
  TT_EMB_SCHED_STEAL_CKPT = 2,
  TT_EMB_SCHED_GROUP = 3
} tt_emb_sched;
tt_emb_status tt_emb_set_schedule(tt_emb_handle h, int mode);

/* Bytes of device workspace for a call with num_indices indices and num_bags
 * bags per table (0 <= num_indices <= desc.max_indices, 0 <= num_bags <=
 * desc.max_bags), at the handle's reuse level; pass the desc maxima for a
 * workspace that serves every call.  The same workspace carries the index
 * grouping from a forward call to the following backward call of the same
 * sizes.  This is the size a backward call (tt_emb_backward,
 * tt_emb_backward_sgd, tt_emb_backward_n) requires; tt_emb_group and the
 * forward calls accept less, since the regions only the backward uses (dE
 * partials and gradient partials) come last in the layout.  Everything
 * bounded by the batch scales with num_indices (about 40 bytes plus 4*D bytes
 * of rows per index, and up to (num_indices/32 + prefix groups) work slices);
 * the dense per-prefix arrays take 12 bytes per (table, i1, i2) slot.  Host
 * only.  TT_EMB_EINVAL for a NULL handle or pointer or sizes out of range. */
tt_emb_status tt_emb_workspace_size(tt_emb_handle h, int64_t num_indices, int64_t num_bags, size_t* bytes);

/* Prefix-based index grouping alone (Section 3.3, Fig. 4): sort the indices
 * of each table, keep exact uniques, take their mixed-radix digits and
 * run-length encode the (i1, i2) prefixes into prefix groups, then order the
 * groups for the fused kernels.  The result stays in `workspace`.  Offsets
 * as described above (NULL = one index per bag). */
tt_emb_status tt_emb_group(tt_emb_handle h, const int64_t* indices, int64_t num_indices, const int64_t* offsets,
                           int64_t num_bags, void* workspace, size_t ws_bytes, void* stream);

/* Forward pass (Section 3.2): out[t][b] = sum over the occurrences o of bag
 * t*B+b of E_{indices[o]}, computed as C = A.B once per prefix group (kept
 * on chip) and E = C.D once per unique row, then sum pooling (an empty bag
 * gives zeros).  `out` is overwritten.  reuse_grouping = 1 skips the
 * grouping step and uses the one already in `workspace` (which must come
 * from a call with the same indices, offsets and sizes on this handle);
 * reuse_grouping = 0 groups first. */
tt_emb_status tt_emb_forward(tt_emb_handle h, const float* G1, const float* G2, const float* G3,
                             const int64_t* indices, int64_t num_indices, const int64_t* offsets, int64_t num_bags,
                             float* out, int reuse_grouping, void* workspace, size_t ws_bytes, void* stream);

/* Forward pass that allocates nothing and takes no workspace, for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation).  It computes what tt_emb_forward
 * with reuse_grouping = 0 computes, with the same kernels, on a workspace held
 * in a static device array of TT_EMB_NOALLOC_SCRATCH_BYTES bytes that each GPU
 * the library runs on keeps until the process ends.  Returns TT_EMB_ESCRATCH,
 * launching nothing, when the call's forward workspace would exceed it (at
 * D = 128 about 100,000 indices fit, less with many prefix slots T*n1*n2).
 * Every call on one GPU shares that GPU's array and leaves its grouping there:
 * calls that overlap on one GPU (other streams or host threads) race and give
 * wrong results; calls in stream order do not.  The grouping it makes is not
 * available to tt_emb_backward (nothing of the caller's workspace is touched).
 * `stream` must belong to the current device (TT_EMB_EINVAL otherwise); at most
 * TT_EMB_NOALLOC_MAX_DEVICES devices.  Other arguments and errors as for
 * tt_emb_forward. */
#define TT_EMB_NOALLOC_SCRATCH_BYTES (64u << 20)
#define TT_EMB_NOALLOC_MAX_DEVICES 64
tt_emb_status tt_emb_forward_noalloc(tt_emb_handle h, const float* G1, const float* G2, const float* G3,
                                     const int64_t* indices, int64_t num_indices, const int64_t* offsets,
                                     int64_t num_bags, float* out, void* stream);

/* Backward pass (Section 3.2, Eq. 1) of L = sum <grad_out, out> into dense
 * core gradients dG1, dG2, dG3 (same shapes as the cores, OVERWRITTEN; rows
 * no index touches are zero).  Per unique row, dE is the sum of grad_out
 * over its occurrences; per row dD = C^T dE and dC = dE D^T; per prefix
 * group the dC are summed first and dA = (sum dC) B^T, dB = A^T (sum dC).
 * The per-core gradients are reduced by segments, with no global float
 * atomics: dG1 is a fixed-order sum of per-slice partials over the slices of
 * each (table, i1), dG2 of per-chunk partials over the chunks of each
 * (table, i2), except on the R = 64 MFMA shape, where each slice's sum dC is
 * kept and dG2 of (table, i2) is the product of the stacked A^T and sum dC of
 * its slices, contracted in slice order.  dG3: on the R = 32 MFMA shape (see
 * tt_emb_kernel_uses_mfma)
 * it is summed in on-chip memory per (table, rank half) and workgroup, then
 * over the workgroups in a fixed order (the on-chip adds land in arrival
 * order, so this dG3 is reproducible to rounding, not bit for bit); on every
 * other shape, the R = 64 MFMA shape included, every unique row's dD is a
 * partial, the rows are put in (table, i3) order by a stable sort, and each
 * dG3 slice is the sum over its rows in that order, so all three gradients
 * are bit-reproducible there.  reuse_grouping as for tt_emb_forward. */
tt_emb_status tt_emb_backward(tt_emb_handle h, const float* G1, const float* G2, const float* G3,
                              const int64_t* indices, int64_t num_indices, const int64_t* offsets,
                              int64_t num_bags, const float* grad_out, float* dG1, float* dG2, float* dG3,
                              int reuse_grouping, void* workspace, size_t ws_bytes, void* stream);

/* Plain SGD step in place on all three cores: G_k -= lr * dG_k (no
 * momentum, no weight decay).  Enqueued on `stream` after the gradients. */
tt_emb_status tt_emb_sgd(tt_emb_handle h, float* G1, float* G2, float* G3, const float* dG1, const float* dG2,
                         const float* dG3, float lr, void* stream);

/* Backward pass and plain SGD in one call: the weight update fused into the
 * backward (an optimisation Section 3.2 describes and leaves out of its
 * final text: each core slice's gradient is aggregated once and applied
 * directly, with no separate optimizer pass).  Leaves every core at
 * G_k - lr * dG_k, with dG_k exactly the gradient tt_emb_backward would
 * return for the same arguments, and writes no gradient arrays.  The update
 * happens after the whole reduction (the kernels that read the cores have
 * finished; rows no index touches are unchanged).  G1..G3 are read and then
 * updated in place; indices, offsets, grad_out, reuse_grouping, workspace
 * and errors as for tt_emb_backward.  The update is applied inside the final
 * segment sums of the gradients, as each element's sum is formed. */
tt_emb_status tt_emb_backward_sgd(tt_emb_handle h, float* G1, float* G2, float* G3, const int64_t* indices,
                                  int64_t num_indices, const int64_t* offsets, int64_t num_bags,
                                  const float* grad_out, float lr, int reuse_grouping, void* workspace,
                                  size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Tables with L TT cores, 2 <= L <= TT_EMB_MAX_CORES.  Eq. 2 splits row g into
 * L mixed-radix digits (i_0, ..., i_{L-1}), i_0 most significant, and the row
 * is the chain of the L core slices: X_0 = S_0, X_k = X_{k-1} . S_k with
 * X_{k-1} viewed as (d_0 ... d_{k-1}) x R, so E = X_{L-1} with output digit
 * j_0 most significant.  The paper names L > 3 as future work; the prefix of
 * Section 3.3 becomes the first L-1 digits.
 *
 * Core k is [T][n_k][r_k][d_k][r_{k+1}] (float32, row-major) with
 * r_0 = r_L = 1 and every other rank R: for L = 3 exactly G1, G2, G3 above.
 * cores and grads are HOST arrays of L device pointers.
 *
 * How the library computes it: for L >= 4 a merged first core
 * [T][n_0...n_{L-3}][d_0...d_{L-3}][R] (the contraction of cores 0..L-3 at
 * every combination of their digits) is built in the workspace at the start
 * of each forward and backward call, one level of the chain at a time (each
 * partial product S_0 ... S_k built once per distinct prefix of k+1 digits),
 * and the three-core operator runs on it and cores L-2, L-1:
 * C = (merged slice) . S_{L-2} once per prefix group of the first L-1 digits,
 * E = C . S_{L-1} per unique row.  The backward carries the merged core's
 * gradient back through the chain one level at a time into cores 0..L-3, each
 * level as per-block partials summed in a fixed order (no atomics).  For L = 2
 * the middle core of the three-core operator is the identity.  Grouping,
 * reuse levels, schedules, errors and tt_emb_debug_grouping work as above on
 * the three-factor view (n_0...n_{L-3}, n_{L-2}, n_{L-1}) for L >= 4 and
 * (n_0, 1, n_1) for L = 2: its digits and prefix keys are those of the view.
 * ---------------------------------------------------------------------- */
#define TT_EMB_MAX_CORES 8

typedef struct {
  int32_t num_tables;                       /* T >= 1 */
  int64_t num_rows;                         /* N, 1 <= N <= n_0 ... n_{L-1} */
  int32_t num_cores;                        /* L, 2 <= L <= TT_EMB_MAX_CORES */
  int32_t row_factors[TT_EMB_MAX_CORES];    /* n_0 .. n_{L-1} >= 1 (entries from L on are ignored) */
  int32_t dim_factors[TT_EMB_MAX_CORES];    /* d_0 .. d_{L-1} >= 1 */
  int32_t rank;                             /* R >= 1 */
  int64_t max_indices;
  int64_t max_bags;
} tt_emb_desc_n;

/* Validate `desc` and create a handle for L cores (host memory only).  The
 * limits of tt_emb_create apply to the three-factor view; in addition
 * n_0 ... n_{L-1} < 2^32 and the merged row product n_0 ... n_{L-3} < 2^28.
 * A handle made here with L = 3 is the same as one from
 * tt_emb_create.  Returns TT_EMB_EINVAL for a bad L, non-positive sizes or
 * N > n_0 ... n_{L-1}, TT_EMB_EUNSUPPORTED beyond the limits.  The three-core
 * calls (tt_emb_forward, tt_emb_backward, tt_emb_backward_sgd, tt_emb_sgd)
 * return TT_EMB_EINVAL on a handle with L != 3; the calls below accept any
 * handle. */
tt_emb_status tt_emb_create_n(const tt_emb_desc_n* desc, tt_emb_handle* out);

/* Forward pass with L cores (Section 3.2 with the chain above): out[t][b] is
 * the sum of the rows of bag t*B+b.  Arguments as for tt_emb_forward; the
 * workspace also holds the merged core (L >= 4; counted by
 * tt_emb_workspace_size).  TT_EMB_EINVAL if cores or any cores[k] is NULL or
 * misaligned. */
tt_emb_status tt_emb_forward_n(tt_emb_handle h, const float* const* cores, const int64_t* indices,
                               int64_t num_indices, const int64_t* offsets, int64_t num_bags, float* out,
                               int reuse_grouping, void* workspace, size_t ws_bytes, void* stream);

/* Backward pass with L cores (Eq. 1 through every product of the chain):
 * grads[k] receives the dense gradient of core k (OVERWRITTEN; rows no index
 * touches are zero).  Arguments as for tt_emb_backward. */
tt_emb_status tt_emb_backward_n(tt_emb_handle h, const float* const* cores, const int64_t* indices,
                                int64_t num_indices, const int64_t* offsets, int64_t num_bags,
                                const float* grad_out, float* const* grads, int reuse_grouping, void* workspace,
                                size_t ws_bytes, void* stream);

/* Plain SGD on the L cores in place: cores[k] -= lr * grads[k]. */
tt_emb_status tt_emb_sgd_n(tt_emb_handle h, float* const* cores, const float* const* grads, float lr,
                           void* stream);

/* Synchronise `stream`, read and clear the sticky device error word of
 * `workspace`.  Returns TT_EMB_OK, TT_EMB_ERANGE or TT_EMB_EHIP. */
tt_emb_status tt_emb_check_errors(tt_emb_handle h, void* workspace, void* stream);

/* Copy the grouping held in `workspace` to host arrays (synchronises
 * `stream`; for tests).  Any output pointer may be NULL.  Sizes: uniq_keys,
 * uniq_digits: U and 3*U; inv: num_indices of the grouped call (-1 for an
 * invalid index); occ_start: U+1; occ_pos: nvalid; pg_start: P+1; pg_keys: P.
 * A unique key is t*(n1*n2*n3) + row; a prefix-group key is t*(n1*n2) +
 * i1*n2 + i2.  counts receives (U, P, nvalid, number of work slices). */
tt_emb_status tt_emb_debug_grouping(tt_emb_handle h, void* workspace, int64_t* uniq_keys, int32_t* uniq_digits,
                                    int32_t* inv, int32_t* occ_start, int32_t* occ_pos, int32_t* pg_start,
                                    int64_t* pg_keys, int64_t* counts, void* stream);

/* Kernels that tt_emb_profile can bracket with events. */
typedef enum {
  TT_EMB_K_NONE = 0,
  TT_EMB_K_INGEST = 1,    /* grouping: keys, positions and bag ids of the occurrences */
  TT_EMB_K_FWD_FUSED = 2, /* forward: C = A.B per prefix group, E = C.D per unique row */
  TT_EMB_K_POOL = 3,      /* forward: sum pooling of E rows into the bags */
  TT_EMB_K_SEG_SUM = 4,   /* backward: dE per unique row, summed over its occurrences */
  TT_EMB_K_BWD_FUSED = 5, /* backward: per prefix group dD, dC, sum dC, dA, dB (dB after it at R = 64) */
  TT_EMB_K_MERGE = 6,     /* L >= 4: merged first core from cores 0..L-3 */
  TT_EMB_K_SPLIT = 7      /* L >= 4 backward: gradients of cores 0..L-3 from the merged core's */
} tt_emb_kernel;

/* Benchmark instrumentation.  While set, every launch of `kernel`
 * (tt_emb_kernel) made through this handle is bracketed by hipEventRecord of
 * ev_begin (a hipEvent_t) before it and ev_end after it, on the stream of the
 * call.  kernel = TT_EMB_K_NONE or NULL events switch it off.  The events
 * stay owned by the caller. */
tt_emb_status tt_emb_profile(tt_emb_handle h, int kernel, void* ev_begin, void* ev_end);

/* Whether `kernel` (TT_EMB_K_FWD_FUSED or TT_EMB_K_BWD_FUSED) runs on the
 * matrix cores for this handle: *uses_mfma = 1 for the MFMA kernels (forward
 * for the view d = (4,4,8) with R = 32 or 64 and for d = (4,4,2) with R = 32;
 * backward for d = (4,4,8) or (4,4,2) with R = 32, n3 <= 252 and at most 64
 * tables, and for d = (4,4,8) with R = 64; all only while
 * their 32-bit offsets into E and the cores fit and, at R = 64, a table's
 * third core spans under 4 GiB), 0 for the generic vector-ALU kernels.
 * Both decide per call from its index count, given here as num_indices
 * (0 <= num_indices <= desc.max_indices).  Every other kernel id reports 0.
 * Host only.
 * TT_EMB_EINVAL for a NULL handle or flag, an unknown kernel id or
 * num_indices out of range. */
tt_emb_status tt_emb_kernel_uses_mfma(tt_emb_handle h, int kernel, int64_t num_indices, int* uses_mfma);

/* Static text for a status code. */
const char* tt_emb_status_string(tt_emb_status s);

#ifdef __cplusplus
}
#endif

#endif /* TT_EMB_H */
