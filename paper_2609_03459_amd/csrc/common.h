// Internal declarations shared by the HIP translation units of libttemb.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ttemb {

constexpr int MAX_CORES = 8;  // largest number of TT cores of a handle

// ---------------------------------------------------------------------------
// Shape and derived constants of one handle.
// ---------------------------------------------------------------------------
struct Shape {
  int T;
  int64_t N;
  int n1, n2, n3;
  int d1, d2, d3;
  int R;
  int D;           // d1*d2*d3
  uint32_t Npad;   // n1*n2*n3: key of (t, g) is t*Npad + g
  uint32_t kinv;   // T*Npad: key given to an invalid occurrence (sorts last)
  int key_bits;    // significant bits of kinv
  int n12;         // n1*n2 prefixes per table
  int64_t ndense;  // T*n1*n2 prefix slots
  int slice_rows;  // rows per work slice: SLICE_ROWS, or 1 when prefix reuse is off (ablation)
  int dedup;       // 1: exact dedup of rows; 0: every occurrence is its own row (ablation)
  int sched;       // work distribution: SCHED_STEAL, SCHED_STATIC, SCHED_STEAL_CKPT or SCHED_GROUP (ablation)
  int chunk_slices;  // slices per chunk of one (t, i2) run (TTEMB_CHUNK, or TTEMB_R64_CHUNK at R = 64)
  // Number of TT cores and their factors.  The fields above are the three-factor
  // view that the grouping and the fused kernels work on: for L = 3 the cores
  // themselves; for L >= 4 (n1, d1) = products of the factors of cores 0..L-3,
  // whose contraction is the merged first core of the view, and (n2, d2),
  // (n3, d3) those of cores L-2 and L-1; for L = 2 (n1, d1) = core 0, a middle
  // identity core with n2 = d2 = 1 and (n3, d3) = core 1.
  int L;
  int nk[MAX_CORES];
  int dk[MAX_CORES];
};

// Counter slots at the head of the workspace (int32).
enum : int {
  C_U = 0,        // unique (table, row) pairs
  C_P = 1,        // prefix groups
  C_NVALID = 2,   // valid occurrences
  C_NSLICES = 3,  // work slices of the fused kernels
  C_ERR = 4,      // sticky error bits
  C_NSEG = 5,     // occurrence chunks of the dE segment sums
  C_NCHUNKS = 8,    // chunks of the specialised kernels
  C_FWD_CTR = 64,         // queue counters of the forward scheduler (stride SCHED_STRIDE)
  C_BWD_CTR = 64 + 4096,  // queue counters of the backward scheduler (stride SCHED_STRIDE)
  C_TOTAL = 64 + 2 * 4096,
};
enum : int { ERR_INDEX = 1, ERR_OFFSETS = 2 };

// Fixed tiling constants.
constexpr int SORT_THREADS = 256;
constexpr int SORT_ITEMS = 16;
constexpr int SORT_TILE = SORT_THREADS * SORT_ITEMS;  // keys per radix tile
constexpr int RADIX_MAX_BITS = 11;               // widest radix digit
constexpr int RADIX_MAX = 1 << RADIX_MAX_BITS;
// LSD radix passes for keys of key_bits bits: equal-width digits of at most RADIX_MAX_BITS
inline int sort_passes(int key_bits) { return (key_bits + RADIX_MAX_BITS - 1) / RADIX_MAX_BITS; }
constexpr int SCAN_THREADS = 256;
constexpr int SCAN_ITEMS = 16;
constexpr int SCAN_TILE = SCAN_THREADS * SCAN_ITEMS;
constexpr int SLICE_ROWS = 32;   // unique rows per work slice
constexpr int CHUNK_SLICES = 32; // most slices per chunk (one (t, i2) run); Shape::chunk_slices <= this
// Slices per chunk at rank 64: the MFMA forward streams B from L2 for every quad
// (nothing is kept per chunk), so short chunks cost no reloads and give the
// persistent waves many more work units than there are waves.
#ifndef TTEMB_R64_CHUNK
#define TTEMB_R64_CHUNK 4
#endif
#ifndef TTEMB_CHUNK
#define TTEMB_CHUNK 32
#endif
constexpr int SEG_CHUNK = 256;   // sorted occurrences per dE chunk
constexpr int MAX_BWD_WG = 256;  // workgroups of the MFMA backward (one per CU on MI355X)

// Device pointers carved out of the caller's workspace.
struct Work {
  int32_t* ctr;           // [C_TOTAL]
  uint32_t* keys[2];      // radix ping-pong keys [M]
  uint32_t* vals[2];      // radix ping-pong positions [M]
  uint32_t* rcounts;      // [RADIX_MAX * ntiles]
  int32_t* tile_bag;      // [ntiles + 1] bag holding the first occurrence of each sort tile
  uint32_t* rtotals;      // [npasses * RADIX_MAX]
  uint64_t* tsum64;       // scan tile sums [ntiles_scan]
  uint32_t* tsum32;       // scan tile sums for 32-bit scans
  int32_t* bag_of;        // [M] global bag of each occurrence
  int32_t* inv;           // [M] unique id of each occurrence (-1 invalid)
  int32_t* sorted_uid;    // [M] unique id of each sorted occurrence
  int32_t* sorted_bag;    // [M] backward: global bag of each sorted occurrence
  uint32_t* uniq_key;     // [M] key of each unique row
  int32_t* uniq_i3;       // [M] last digit i3 of each unique row
  int32_t* occ_start;     // [M+1] first sorted position of each unique row
  int32_t* pg_start;      // [M+1] first unique row of each prefix group
  uint32_t* pg_key;       // [M] t*n1*n2 + i1*n2 + i2 of each group
  uint32_t* dense_cnt;    // [ndense] slices per prefix slot, (t, i2, i1) order
  uint32_t* dense_base;   // [ndense] exclusive scan of dense_cnt
  int32_t* dense_pg;      // [ndense] group id per slot
  int4* slices;           // [nsl_max] (group, row_begin, row_end, key)
  int32_t* slice_i1;      // [nsl_max] first digit i1 of each slice's group
  uint32_t* run_nch;      // [T*n2 + 1] chunks per (t, i2) run, then their exclusive scan
  int4* chunks;           // [nch_max] (first slice, slice count, run, 0)
  float* dApart;          // backward: dA of each slice, [2][nsl_max][d1*R] (MFMA: one per rank half) or
                          // [nsl_max][d1*R] (generic)
  float* dBpart;          // backward: dB of each chunk, [2][nch_max][R*d2*R/2] (R = 32 MFMA) or [nch_max][R*d2*R]
                          // (generic); null on the R = 64 MFMA path, which keeps dCpart instead
  float* dCpart;          // R = 64 MFMA backward: dC sum of each slice, [nsl_max][d1][d2*R]
  float* g3part;          // [MAX_BWD_WG][n3*R*d3/2] backward: dG3 half of each workgroup
  // generic backward (shapes the MFMA backward does not serve), else null: partials of
  // the fixed-order segment sums and the (table, i3) order of the unique rows
  float* dDpart;          // [M][R*d3] dD of each unique row
  uint32_t* g3keys[2];    // [M] sort keys t*n3 + i3 of the unique rows (ping-pong)
  uint32_t* g3vals[2];    // [M] unique row ids (ping-pong)
  int32_t* g3lo;          // [T*n3] first position of each (t, i3) in the sorted rows
  int32_t* g3hi;          // [T*n3] one past its last
  float* g1m;             // L >= 4: merged first core [T][n1][d1][R] of the view; L = 2: identity middle core
                          // [T][1][R][1][R]; null for L = 3
  float* dg1m;            // gradient of g1m (same size; for L = 2 computed and discarded)
  float* xlev;            // L >= 5: partial products of the merged cores' inner levels, chain_level_floats(s)
  float* dxlev;           // L >= 5: their gradients (same size)
  float* splitpart;       // L >= 4: partials of one backward level of the merged chain, split_partial_floats(s)
  float* ckpt;            // [CKPT_SLOTS][d1*d2*R] checkpointed C of the generic kernels (null for the MFMA shape)
  int32_t* ckpt_tag;      // [CKPT_SLOTS] prefix group held by each entry, -1 = none
  int64_t nsl_max, nch_max;
  float* E;               // [M][D]: E rows (forward), dE rows (backward)
  float* seg_part;        // [nseg][2][D] partial dE of rows that cross a chunk
  uint32_t* sorted_keys;  // = keys[x] after the sort
  uint32_t* sorted_pos;   // = vals[x] after the sort
  int64_t M;              // capacity in occurrences
  int64_t B;              // capacity in bags per table
};

// Event bracketing of one kernel for benchmarks (ids of tt_emb_kernel).
struct Prof {
  int kernel;
  hipEvent_t begin, end;
};
enum : int { K_INGEST = 1, K_FWD_FUSED = 2, K_POOL = 3, K_SEG_SUM = 4, K_BWD_FUSED = 5, K_MERGE = 6, K_SPLIT = 7 };
inline void prof_begin(const Prof& p, int k, hipStream_t st) {
  if (p.kernel == k && p.begin) (void)hipEventRecord(p.begin, st);
}
inline void prof_end(const Prof& p, int k, hipStream_t st) {
  if (p.kernel == k && p.end) (void)hipEventRecord(p.end, st);
}

// Workspace layout for given capacities (bytes) and carving.
size_t workspace_bytes(const Shape& s, int64_t M, int64_t B);
// Bytes of that layout a forward call uses (the regions before the backward-only ones).
size_t forward_workspace_bytes(const Shape& s, int64_t M, int64_t B);
void carve(const Shape& s, int64_t M, int64_t B, void* base, Work* w);

// Launchers (each returns hipGetLastError() of its launches).
hipError_t launch_group(const Shape& s, const Work& w, const int64_t* idx, int64_t M, const int64_t* offsets,
                        int64_t B, const Prof& prof, hipStream_t st);
hipError_t launch_forward(const Shape& s, const Work& w, const float* G1, const float* G2, const float* G3,
                          const int64_t* offsets, int64_t M, int64_t B, float* out, const Prof& prof,
                          hipStream_t st);
// With update set, dG1..dG3 are the cores and receive G -= lr * dG (no gradient arrays written).
hipError_t launch_backward(const Shape& s, const Work& w, const float* G1, const float* G2, const float* G3,
                           const int64_t* offsets, int64_t M, int64_t B, const float* dV, float* dG1, float* dG2,
                           float* dG3, float lr, bool update, const Prof& prof, hipStream_t st);
hipError_t launch_sgd(const Shape& s, float* G1, float* G2, float* G3, const float* dG1, const float* dG2,
                      const float* dG3, float lr, hipStream_t st);
// L-core handles (cores.hip).  cores[k] / grads[k] are the device arrays of core k.
// Merged first core of the view from cores 0..L-3 (L >= 4), level by level, into w.g1m.
hipError_t launch_merge(const Shape& s, const Work& w, const float* const* cores, const Prof& prof, hipStream_t st);
// Gradients of cores 0..L-3 from the merged core's gradient w.dg1m (L >= 4), level by level
// (reads the levels launch_merge left in w; overwrites the gradients).
hipError_t launch_split(const Shape& s, const Work& w, const float* const* cores, float* const* grads,
                        const Prof& prof, hipStream_t st);
// Identity middle core of an L = 2 handle, into w.g1m.
hipError_t launch_identity(const Shape& s, const Work& w, hipStream_t st);
// Element count of core k.
int64_t core_elems(const Shape& s, int k);
// Floats of the inner partial-product levels of the merged cores (0 when L < 5).
int64_t chain_level_floats(const Shape& s);
// Floats of the largest level's partials in the backward of the merged chain (0 when L < 4).
int64_t split_partial_floats(const Shape& s);
// G -= lr * dG on n floats.
hipError_t launch_sgd1(float* G, const float* dG, int64_t n, float lr, hipStream_t st);
// Whether the MFMA backward (and its partial-sum workspace) serves this shape.
bool bwd_r32_supported(const Shape& s, int64_t max_indices);
// Whether the MFMA backward for R = 64 serves this shape (it writes the generic
// backward's partials, so needs no workspace of its own).
bool bwd_r64_supported(const Shape& s, int64_t max_indices);
// Whether the MFMA forward serves this shape (R = 32, R = 64).
bool fwd_r32_supported(const Shape& s, int64_t max_indices);
bool fwd_r64_supported(const Shape& s, int64_t max_indices);

// Stable radix sort of n pairs between keys[0..1] / vals[0..1] (input in index 0); *out
// = the index holding the result (group.hip).
hipError_t sort_pairs(const Work& w, uint32_t* const keys[2], uint32_t* const vals[2], int n, int key_bits,
                      int* out, hipStream_t st);

// Small generic kernels shared across units (defined in group.hip).
hipError_t fill_u32(uint32_t* p, int64_t n, uint32_t v, hipStream_t st);
hipError_t fill_f32(float* p, int64_t n, float v, hipStream_t st);
hipError_t scan_u32_exclusive(const uint32_t* in, uint32_t* out, int64_t n, uint32_t* tsum, int32_t* total_out,
                              hipStream_t st);
int persistent_grid();

// The dispatcher deals workgroups to the eight XCDs in turn (XCD = block id mod 8),
// and each XCD has its own L2.  A launch of xcd_grid(n) blocks that takes its work
// item from xcd_block gives every XCD one contiguous eighth of the items, so data
// that neighbouring items share (rows of one table) is cached in one L2.  Items
// past n land on the last blocks and must be skipped by the kernel.
constexpr unsigned NUM_XCD = 8;
inline unsigned xcd_grid(unsigned n) { return (n + NUM_XCD - 1) / NUM_XCD * NUM_XCD; }
__device__ __forceinline__ unsigned xcd_block(unsigned b, unsigned grid) {
  return (b % NUM_XCD) * (grid / NUM_XCD) + b / NUM_XCD;
}

// ---------------------------------------------------------------------------
// Device helpers.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }
// the value of lane L ^ 1 (DPP quad permutation 1, 0, 3, 2)
__device__ __forceinline__ float swap_neighbour(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0xB1, 0xF, 0xF, false));
}

template <typename T>
__device__ __forceinline__ T wave_incl_scan(T v) {
  const int lane = lane_id();
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    T u = __shfl_up(v, o, 64);
    if (lane >= o) v += u;
  }
  return v;
}

// Exclusive scan over a block of NT threads; smem holds NT/64 values.
template <typename T, int NT>
__device__ __forceinline__ T block_excl_scan(T v, T* smem, T* total) {
  constexpr int NW = NT / 64;
  T inc = wave_incl_scan(v);
  const int w = threadIdx.x >> 6;
  if (lane_id() == 63) smem[w] = inc;
  __syncthreads();
  T base = 0, tot = 0;
#pragma unroll
  for (int k = 0; k < NW; ++k) {
    T x = smem[k];
    if (k < w) base += x;
    tot += x;
  }
  __syncthreads();
  *total = tot;
  return base + inc - v;
}

}  // namespace ttemb

namespace ttemb {

// Cache policy of arrays that one kernel writes and a later kernel reads.  Partial
// results that a reduction reads exactly once are loaded non-temporally there, and
// the backward's dA, dB and dC partials are also stored non-temporally.  Embedding rows,
// dE and the per-row dD partials are stored non-temporally when the array is larger
// than the chip's 256 MB last-level cache (MALL): it cannot stay there for its reader,
// and ordinary stores would push out lines the writer itself still reads; smaller
// ones are stored normally, so that their reader finds them in that cache.
constexpr uint64_t STREAM_BYTES = 256ull << 20;
constexpr int CPOL_NT = 2;  // buffer-store cache policy: non-temporal
__device__ __forceinline__ float ntl(const float* p) { return __builtin_nontemporal_load(p); }
__device__ __forceinline__ float2 ntl2(const float2* p) {
  typedef float f32x2v __attribute__((ext_vector_type(2)));
  const f32x2v v = __builtin_nontemporal_load(reinterpret_cast<const f32x2v*>(p));
  return make_float2(v.x, v.y);
}

// Persistent-thread scheduler with chunked work stealing (FlowTT Section 3.4).
// The chunk list is cut into nq contiguous queues; queue v holds chunks
// [share_lo(v), share_lo(v + 1)) and has one claim counter on a 128-byte line
// of its own.  A worker claims the next chunk of its home queue with a single
// atomic (consecutive chunks, so neighbouring groups stay in the home XCD's L2);
// once the home queue is empty it steals from the following queues in turn.  An
// empty queue is never visited again, so a worker makes at most nq failed
// claims before it exits.  The forward uses one queue per XCD (workgroup
// blockIdx % 8 runs on XCD blockIdx % 8); the specialised backward gives every
// (table, rank half) owner one queue, since its LDS accumulator is its own.
constexpr int SCHED_NQ = 8;       // queues of the forward scheduler: one per XCD
constexpr int SCHED_STRIDE = 32;  // ints between queue counters (128 bytes)

__device__ __forceinline__ int share_lo(int nchunks, int W, int v) { return (int)(((int64_t)nchunks * v) / W); }

__device__ __forceinline__ int claim_queues(int32_t* q, int nchunks, int nq, int home, int* cursor) {
  while (*cursor < nq) {
    int v = home + *cursor;
    if (v >= nq) v -= nq;
    const int lo = share_lo(nchunks, nq, v), hi = share_lo(nchunks, nq, v + 1);
    int c = -1;
    if (lane_id() == 0) {
      const int got = atomicAdd(&q[v * SCHED_STRIDE], 1);
      if (lo + got < hi) c = lo + got;
    }
    c = __builtin_amdgcn_readfirstlane(c);
    if (c >= 0) return c;
    ++*cursor;
  }
  return -1;
}

// Block-level worker: wave 0 claims for the block.
__device__ __forceinline__ int claim_block(int32_t* q, int nchunks, int nq, int home, int* cursor, int* s_chunk) {
  if (threadIdx.x < 64) {
    const int c = claim_queues(q, nchunks, nq, home, cursor);
    if (threadIdx.x == 0) *s_chunk = c;
  }
  __syncthreads();
  int c = *s_chunk;
  __syncthreads();
  return c;
}

// Work distribution modes (values of the C-ABI's tt_emb_sched).
enum : int { SCHED_STEAL = 0, SCHED_STATIC = 1, SCHED_STEAL_CKPT = 2, SCHED_GROUP = 3 };
// Static modes: fixed contiguous shares of the chunk list (SCHED_GROUP: chunks are
// whole prefix groups, see GROUP_CHUNK_MAX).
__host__ __device__ __forceinline__ bool sched_static(int sched) { return sched == SCHED_STATIC || sched == SCHED_GROUP; }
// SCHED_GROUP cuts chunks at prefix-group boundaries: one chunk per group, a group
// of more slices than this (more than 2,048 rows) in pieces of this many, which the
// fused kernels' per-lane slice descriptors bound.
constexpr int GROUP_CHUNK_MAX = 64;
// Checkpoint table of the generic fused kernels: CKPT_SLOTS entries of one C
// (d1 d2 R floats) each, tagged with the prefix group they hold.
constexpr int CKPT_SLOTS = 1024;

// The next chunk of a block-level worker: its fixed contiguous share in order
// (SCHED_STATIC; *next starts at the share's first chunk), or from the shared
// queues with stealing.  `sched` is a kernel argument, so every thread of the
// block takes the same branch.
__device__ __forceinline__ int claim_block_sched(int sched, int32_t* q, int nchunks, int home, int* cursor,
                                                 int* s_chunk, int* next) {
  if (sched_static(sched)) {
    const int hi = share_lo(nchunks, (int)gridDim.x, (int)blockIdx.x + 1);
    return *next < hi ? (*next)++ : -1;
  }
  return claim_block(q, nchunks, SCHED_NQ, home, cursor, s_chunk);
}

// Checkpointed intermediates of the generic kernels (Section 3.5).  The entry of
// prefix group p is slot p mod CKPT_SLOTS; its tag holds p when complete, CKPT_BUSY
// while a block writes it and CKPT_EMPTY after the per-launch reset.  A writer
// first swaps the tag to CKPT_BUSY (so writers of one slot exclude each other) and
// publishes p after the data; a reader accepts the data only if the tag read p
// both before and after its copy.
constexpr int32_t CKPT_BUSY = -1, CKPT_EMPTY = -2;

// Block-wide: copies p's checkpoint into C (nC floats, LDS) and returns true, or
// returns false (C unspecified) when the entry does not hold p.
__device__ __forceinline__ bool ckpt_load(const float* ckpt, int32_t* tag, int p, float* C, int nC, int* s_flag) {
  const int slot = p % CKPT_SLOTS;
  if (threadIdx.x == 0)
    *s_flag = __hip_atomic_load(tag + slot, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT) == p;
  __syncthreads();
  const bool hit = *s_flag;
  __syncthreads();
  if (!hit) return false;
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  const float* src = ckpt + (size_t)slot * nC;
  for (int o = threadIdx.x; o < nC; o += blockDim.x) C[o] = __builtin_nontemporal_load(src + o);
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  __syncthreads();
  if (threadIdx.x == 0)
    *s_flag = __hip_atomic_load(tag + slot, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT) == p;
  __syncthreads();
  const bool still = *s_flag;
  __syncthreads();
  return still;
}

// Block-wide: publishes C (nC floats, LDS) as p's checkpoint unless another block
// is writing that slot.
__device__ __forceinline__ void ckpt_store(float* ckpt, int32_t* tag, int p, const float* C, int nC, int* s_flag) {
  const int slot = p % CKPT_SLOTS;
  if (threadIdx.x == 0) {
    int32_t seen = __hip_atomic_load(tag + slot, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    *s_flag = seen != CKPT_BUSY &&
              __hip_atomic_compare_exchange_strong(tag + slot, &seen, CKPT_BUSY, __ATOMIC_ACQ_REL,
                                                   __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();
  const bool mine = *s_flag;
  __syncthreads();
  if (!mine) return;
  float* dst = ckpt + (size_t)slot * nC;
  for (int o = threadIdx.x; o < nC; o += blockDim.x) dst[o] = C[o];
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
  __syncthreads();
  if (threadIdx.x == 0) __hip_atomic_store(tag + slot, p, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
}

struct ShapeArgs {  // shape constants passed by value to kernels
  int T, n1, n2, n3, d1, d2, d3, R, D, n12;
  uint32_t Npad;
  int sched;
};


}  // namespace ttemb

namespace ttemb {

// Digits of a sorted key t*Npad + g (Eq. 2: i1 = g / (n2 n3), i2 = (g / n3) mod n2,
// i3 = g mod n3); every kernel decodes keys through this one function.
struct Digits {
  int t, i1, i2, i3;
};
__device__ __forceinline__ Digits decode_key(uint32_t key, uint32_t Npad, int n2, int n3) {
  Digits d;
  d.t = (int)(key / Npad);
  const uint32_t g = key - (uint32_t)d.t * Npad;
  const uint32_t q = g / (uint32_t)n3;
  d.i3 = (int)(g - q * (uint32_t)n3);
  d.i1 = (int)(q / (uint32_t)n2);
  d.i2 = (int)(q - (uint32_t)d.i1 * (uint32_t)n2);
  return d;
}

hipError_t launch_debug_digits(const Shape& s, const Work& w, int32_t* out, int U, int which, hipStream_t st);

}  // namespace ttemb

namespace ttemb {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// one of four wave-uniform values by a per-lane index
template <typename T>
__device__ __forceinline__ T sel4(int j, T a, T b, T c, T d) {
  return j == 0 ? a : (j == 1 ? b : (j == 2 ? c : d));
}

// Raw buffer loads through a gfx9 buffer descriptor (stride 0, dword data):
// the address is base + offset (+ a wave-uniform offset), and a load at or past
// num_bytes returns zero instead of touching memory.
typedef __amdgpu_buffer_rsrc_t buf_t;
__device__ __forceinline__ buf_t make_buf(const void* base, uint32_t num_bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)num_bytes, 0x00020000);
}
__device__ __forceinline__ float buf_f32(buf_t r, uint32_t off, uint32_t soff = 0) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, soff, 0));
}
__device__ __forceinline__ float2 buf_f32x2(buf_t r, uint32_t off) {
  return __builtin_bit_cast(float2, __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0));
}
__device__ __forceinline__ float4 buf_f32x4(buf_t r, uint32_t off) {
  return __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}

// Waits until every vector memory access of this wave has completed (s_waitcnt
// vmcnt(0), the other counters untouched: expcnt 7, lgkmcnt 15).  The compiler
// keeps such an explicit wait and counts it when it places its own waits.
__device__ __forceinline__ void vm_wait_all() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Orders this wave's LDS writes before its later LDS reads of other lanes'
// data (a wave's LDS requests complete in order; this keeps the compiler
// from reordering across the exchange and waits for outstanding writes).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

}  // namespace ttemb
