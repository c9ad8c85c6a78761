// Backward pass of the TT-embedding gather (FlowTT Section 3.2, Eq. 1) and SGD.
//   dE segment sums : dE_u = sum of grad_out rows over the occurrences of u,
//                     walked in sorted order in fixed chunks; a short row that
//                     crosses a chunk end is summed whole by its first chunk,
//                     a long one is finished from per-chunk partials
//                     (deterministic, no atomics)
//   per group       : C recomputed, dD_u = C^T dE_u and dC_u = dE_u D_u^T per row,
//                     sum dC over the group first, then dA = (sum dC) B^T and
//                     dB = A^T (sum dC)
#include "common.h"

namespace ttemb {

ShapeArgs shape_args(const Shape& s);
hipError_t launch_bwd_r64(const Shape& s, const Work& w, const float* G1, const float* G2, const float* G3,
                          const Prof& prof, hipStream_t st);
hipError_t launch_dg2_r64(const Shape& s, const Work& w, const float* G1, float* dG2, float lr, bool update,
                          hipStream_t st);
hipError_t launch_bwd_r32(const Shape& s, const Work& w, const float* G1, const float* G2, const float* G3,
                          float* dG1, float* dG2, float* dG3, float lr, bool update, const Prof& prof,
                          hipStream_t st);

// ---------------------------------------------------------------------------
// dE segment sums over the sorted occurrences
// ---------------------------------------------------------------------------
// What chunk c = [i0, i1) of the sorted occurrences sums.  A row's occurrences
// are contiguous, so only the chunk's first row can have begun before it and only
// its last row can go on after it.  A row of at most SEG_CHUNK occurrences that
// crosses the chunk end is summed whole by the chunk of its first occurrence,
// which reads on past its end (less than one chunk), and skipped by the next
// chunk.  A longer row is split: each chunk sums its part into a partial (head:
// the row began in an earlier chunk; tail: it goes on after this one), and
// k_seg_fix adds the parts.
struct SegEnds {
  int ib, ie;            // occurrences summed here: [ib, ie), empty when ib >= ie
  int u_head, u_tail;    // the rows whose sums go to the head / tail partial, else -1
};
__device__ __forceinline__ SegEnds seg_ends(const int32_t* __restrict__ sorted_uid,
                                            const int32_t* __restrict__ occ_start, int i0, int i1, int nvalid) {
  SegEnds e;
  e.ib = i0;
  e.ie = i1;
  e.u_head = e.u_tail = -1;
  const int uf = sorted_uid[i0];
  if (i0 > 0 && sorted_uid[i0 - 1] == uf) {
    const int end = occ_start[uf + 1];
    if (end - occ_start[uf] <= SEG_CHUNK)
      e.ib = end;  // summed by the previous chunk
    else
      e.u_head = uf;
  }
  const int ul = sorted_uid[i1 - 1];
  if (i1 < nvalid && sorted_uid[i1] == ul) {
    const int end = occ_start[ul + 1];
    if (end - occ_start[ul] <= SEG_CHUNK)
      e.ie = end;  // read on to the row's end
    else if (ul != e.u_head)
      e.u_tail = ul;
  }
  return e;
}
__device__ __forceinline__ float* seg_dst(const SegEnds& e, int cur, int c, int D, float* __restrict__ dE,
                                          float* __restrict__ part) {
  if (cur == e.u_head) return part + ((int64_t)c * 2 + 0) * D;
  if (cur == e.u_tail) return part + ((int64_t)c * 2 + 1) * D;
  return dE + (int64_t)cur * D;
}
__device__ __forceinline__ void seg_flush(const SegEnds& e, int cur, int c, int D, int j0, const float* acc,
                                          float* __restrict__ dE, float* __restrict__ part) {
  float* dst = seg_dst(e, cur, c, D, dE, part);
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int j = j0 + k * 64 + lane_id();
    if (j < D) dst[j] = acc[k];
  }
}

// The bag of every sorted occurrence, gathered once through the sorted positions,
// so that the dE sums read it in order instead of chasing two indices per row.
// Blocks take contiguous runs of SB_ITEMS x 256 sorted occurrences, an eighth of
// them per XCD: the sorted order is table by table, so an XCD reads the bag ids of
// about one table, a range its L2 holds.
constexpr int SB_ITEMS = 4;
__global__ void __launch_bounds__(256) k_sorted_bag(const uint32_t* __restrict__ sorted_pos,
                                                    const int32_t* __restrict__ bag_of,
                                                    const int32_t* __restrict__ ctr, int32_t* __restrict__ sorted_bag) {
  const int nvalid = ctr[C_NVALID];
  const int i0 = (int)xcd_block(blockIdx.x, gridDim.x) * (SB_ITEMS * 256) + (int)threadIdx.x;
  uint32_t p[SB_ITEMS];
#pragma unroll
  for (int k = 0; k < SB_ITEMS; ++k) p[k] = i0 + 256 * k < nvalid ? sorted_pos[i0 + 256 * k] : 0u;
  int32_t b[SB_ITEMS];
#pragma unroll
  for (int k = 0; k < SB_ITEMS; ++k) b[k] = i0 + 256 * k < nvalid ? bag_of[p[k]] : 0;
#pragma unroll
  for (int k = 0; k < SB_ITEMS; ++k)
    if (i0 + 256 * k < nvalid) sorted_bag[i0 + 256 * k] = b[k];
}

// One wave per chunk of SEG_CHUNK sorted occurrences; lanes hold 4 columns
// each (column blocks of 256); occurrence indices are fetched 64 at a time and
// the grad_out rows of 8 occurrences are loaded before they are summed.
// Four waves per workgroup (one-wave workgroups would cap the waves a CU holds),
// each wave one chunk.
constexpr int SEG_WAVES = 4;

__global__ void __launch_bounds__(64 * SEG_WAVES) k_seg_dE(const float* __restrict__ dV, const int32_t* __restrict__ sorted_uid,
                                               const int32_t* __restrict__ sorted_bag,
                                               const int32_t* __restrict__ occ_start,
                                               const int32_t* __restrict__ ctr, int D, float* __restrict__ dE,
                                               float* __restrict__ part) {
  const int nvalid = ctr[C_NVALID];
  const int c = blockIdx.x * SEG_WAVES + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int i0 = c * SEG_CHUNK;
  if (i0 >= nvalid) return;
  const int lane = lane_id();
  const SegEnds ends = seg_ends(sorted_uid, occ_start, i0, i0 + SEG_CHUNK < nvalid ? i0 + SEG_CHUNK : nvalid, nvalid);
  const int ib = ends.ib, ie = ends.ie;
  if (ib >= ie) return;
  for (int j0 = 0; j0 < D; j0 += 256) {
    bool colok[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) colok[q] = j0 + q * 64 + lane < D;
    int cur = sorted_uid[ib];
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    for (int base = ib; base < ie; base += 64) {
      const int i = base + lane;
      const int my_u = i < ie ? sorted_uid[i] : -1;
      const int my_b = i < ie ? sorted_bag[i] : 0;
      const int cnt = ie - base < 64 ? ie - base : 64;
      for (int k0 = 0; k0 < cnt; k0 += 8) {
        float v[8][4];
        int uk[8];
#pragma unroll
        for (int kk = 0; kk < 8; ++kk) {
          const int k = k0 + kk < cnt ? k0 + kk : k0;
          const int b = __shfl(my_b, k, 64);
          uk[kk] = __shfl(my_u, k, 64);
          const float* row = dV + (int64_t)b * D + j0 + lane;
#pragma unroll
          for (int q = 0; q < 4; ++q) v[kk][q] = colok[q] ? row[q * 64] : 0.f;
        }
#pragma unroll
        for (int kk = 0; kk < 8; ++kk) {
          if (k0 + kk < cnt) {
            if (uk[kk] != cur) {
              seg_flush(ends, cur, c, D, j0, acc, dE, part);
              cur = uk[kk];
              acc[0] = acc[1] = acc[2] = acc[3] = 0.f;
            }
#pragma unroll
            for (int q = 0; q < 4; ++q) acc[q] += v[kk][q];
          }
        }
      }
    }
    seg_flush(ends, cur, c, D, j0, acc, dE, part);
  }
}

// D = 128 and D = 32: a lane owns two columns (one 8-byte load per occurrence;
// for D = 32 sixteen lanes cover a row and the other lanes repeat their loads),
// the bag index of each occurrence is read into a scalar register so every dV row
// is a uniform base, and 16 (D = 128) or 32 (D = 32) rows are in flight before
// they are summed in order.  Chunks go in sorted order, an eighth of them per XCD,
// so each XCD reads the grad_out rows and bag ids of about one table, and more of
// them hit its L2.
template <int D>
__device__ __forceinline__ void seg_rows(const float* __restrict__ dV, const int32_t* __restrict__ sorted_uid,
                                         const int32_t* __restrict__ sorted_bag, const int32_t* __restrict__ occ_start,
                                         const int32_t* __restrict__ ctr, float* __restrict__ dE,
                                         float* __restrict__ part) {
  constexpr int LN = D / 2;               // lanes that own columns
  constexpr int KB = D == 128 ? 16 : 32;  // rows in flight
  const int nvalid = ctr[C_NVALID];
  const int c = (int)xcd_block(blockIdx.x, gridDim.x) * SEG_WAVES + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int i0 = c * SEG_CHUNK;
  if (i0 >= nvalid) return;  // also the blocks past the chunk count that round the grid to 8
  const int lane = lane_id();
  const int col = lane % LN;
  const SegEnds ends = seg_ends(sorted_uid, occ_start, i0, i0 + SEG_CHUNK < nvalid ? i0 + SEG_CHUNK : nvalid, nvalid);
  const int ib = ends.ib, ie = ends.ie;
  if (ib >= ie) return;
  // dE of all unique rows beyond the last-level cache: stored non-temporally.  The row
  // goes through a descriptor of its 4 D bytes (lanes past LN fall outside it), so the
  // two cache policies stay two distinct stores
  const bool de_nt = (uint64_t)(uint32_t)ctr[C_U] * (4u * D) > STREAM_BYTES;
  auto flush = [&](int u, float2 acc) {
    typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
    const buf_t row = make_buf(seg_dst(ends, u, c, D, dE, part), 4u * D);
    const u32x2 v = u32x2{__float_as_uint(acc.x), __float_as_uint(acc.y)};
    if (de_nt)
      __builtin_amdgcn_raw_buffer_store_b64(v, row, 8u * (uint32_t)lane, 0, CPOL_NT);
    else
      __builtin_amdgcn_raw_buffer_store_b64(v, row, 8u * (uint32_t)lane, 0, 0);
  };
  int cur = sorted_uid[ib];
  float2 acc = make_float2(0.f, 0.f);
  for (int base = ib; base < ie; base += 64) {
    const int i = base + lane;
    const int my_u = i < ie ? sorted_uid[i] : -1;
    const int my_b = i < ie ? sorted_bag[i] : 0;
    const int cnt = ie - base < 64 ? ie - base : 64;
    for (int k0 = 0; k0 < cnt; k0 += KB) {
      float2 v[KB];
#pragma unroll
      for (int kk = 0; kk < KB; ++kk) {
        const int k = k0 + kk < cnt ? k0 + kk : k0;  // clamped: every load is unconditional
        const int b = __builtin_amdgcn_readlane(my_b, k);
        v[kk] = reinterpret_cast<const float2*>(dV + (size_t)b * D)[col];
      }
#pragma unroll
      for (int kk = 0; kk < KB; ++kk) {
        if (k0 + kk < cnt) {
          const int u = __builtin_amdgcn_readlane(my_u, k0 + kk);
          if (u != cur) {
            flush(cur, acc);
            cur = u;
            acc = make_float2(0.f, 0.f);
          }
          acc.x += v[kk].x;
          acc.y += v[kk].y;
        }
      }
    }
  }
  flush(cur, acc);
}
__global__ void __launch_bounds__(64 * SEG_WAVES) k_seg_dE128(const float* __restrict__ dV, const int32_t* __restrict__ sorted_uid,
                                                  const int32_t* __restrict__ sorted_bag,
                                                  const int32_t* __restrict__ occ_start,
                                                  const int32_t* __restrict__ ctr, float* __restrict__ dE,
                                                  float* __restrict__ part) {
  seg_rows<128>(dV, sorted_uid, sorted_bag, occ_start, ctr, dE, part);
}
__global__ void __launch_bounds__(64 * SEG_WAVES) k_seg_dE32(const float* __restrict__ dV, const int32_t* __restrict__ sorted_uid,
                                                 const int32_t* __restrict__ sorted_bag,
                                                 const int32_t* __restrict__ occ_start,
                                                 const int32_t* __restrict__ ctr, float* __restrict__ dE,
                                                 float* __restrict__ part) {
  seg_rows<32>(dV, sorted_uid, sorted_bag, occ_start, ctr, dE, part);
}

// Rows of more than SEG_CHUNK occurrences: chunk c0 + 1, where c0 holds the
// row's first occurrence, finishes the row from c0's tail partial and the head
// partials of every following chunk, in chunk order.  A block screens 64 chunks
// with one lane each (few of them start inside such a row).  Rows of at most
// FIX_SMALL head partials are fixed one per wave, all at once; longer rows one
// after the other by the whole block: its waves split the chunk range, each
// sums its part with four independent accumulators per column, and the parts
// are combined in a fixed order.
constexpr int FIX_SCREEN = 64;  // chunks screened per block
constexpr int FIX_WAVES = 16;
constexpr int FIX_SMALL = 16;
__device__ __forceinline__ int fix_row(const int32_t* __restrict__ sorted_uid, const int32_t* __restrict__ occ_start,
                                       int c, int* c0, int* c1) {
  const int u = sorted_uid[c * SEG_CHUNK];
  const int lo = occ_start[u], hi = occ_start[u + 1];
  *c0 = lo / SEG_CHUNK;
  *c1 = (hi - 1) / SEG_CHUNK;
  return u;
}
__global__ void __launch_bounds__(64 * FIX_WAVES) k_seg_fix(const int32_t* __restrict__ sorted_uid,
                                                            const int32_t* __restrict__ occ_start,
                                                            const int32_t* __restrict__ ctr, int D,
                                                            const float* __restrict__ part, float* __restrict__ dE) {
  __shared__ float red[FIX_WAVES][256];
  __shared__ uint64_t flagged[2];  // rows with few / many head partials
  const int nvalid = ctr[C_NVALID];
  const int w = threadIdx.x >> 6, lane = lane_id();
  if (w == 0) {
    const int c = blockIdx.x * FIX_SCREEN + lane;
    bool fix = false, big = false;
    if (c > 0 && (int64_t)c * SEG_CHUNK < nvalid) {
      const int u = sorted_uid[c * SEG_CHUNK];
      const int lo = occ_start[u], hi = occ_start[u + 1];
      fix = lo / SEG_CHUNK == c - 1 && hi - lo > SEG_CHUNK;
      big = (hi - 1) / SEG_CHUNK - lo / SEG_CHUNK > FIX_SMALL;
    }
    const uint64_t m_small = __ballot(fix && !big), m_big = __ballot(fix && big);
    if (lane == 0) {
      flagged[0] = m_small;
      flagged[1] = m_big;
    }
  }
  __syncthreads();
  // short rows: the v-th flagged chunk goes to wave v mod FIX_WAVES
  {
    uint64_t m = flagged[0];
    for (int v = 0; m; ++v, m &= m - 1) {
      if (v % FIX_WAVES != w) continue;
      int c0, c1;
      const int u = fix_row(sorted_uid, occ_start, blockIdx.x * FIX_SCREEN + __builtin_ctzll(m), &c0, &c1);
      for (int j = lane; j < D; j += 64) {
        float a[4] = {part[((int64_t)c0 * 2 + 1) * D + j], 0.f, 0.f, 0.f};
        int k = c0 + 1;
        for (; k + 4 <= c1 + 1; k += 4)
#pragma unroll
          for (int kk = 0; kk < 4; ++kk) a[kk] += part[((int64_t)(k + kk) * 2 + 0) * D + j];
        for (; k <= c1; ++k) a[0] += part[((int64_t)k * 2 + 0) * D + j];
        dE[(int64_t)u * D + j] = (a[0] + a[1]) + (a[2] + a[3]);
      }
    }
  }
  // long rows: the whole block on each
  uint64_t m = flagged[1];
  while (m) {
    const int c = blockIdx.x * FIX_SCREEN + __builtin_ctzll(m);
    m &= m - 1;
    int c0, c1;
    const int u = fix_row(sorted_uid, occ_start, c, &c0, &c1);
    const int n = c1 - c0;  // head partials of chunks c0+1 .. c1
    const int k_lo = c0 + 1 + (int)(((int64_t)n * w) / FIX_WAVES);
    const int k_hi = c0 + 1 + (int)(((int64_t)n * (w + 1)) / FIX_WAVES);
    if ((D & 1) == 0 && D <= 128) {
      // a lane owns a column pair, so one load takes a whole partial row, and eight
      // partials are in flight per wave
      const int jc = 2 * lane;
      const bool ok = jc < D;
      float2 a[8];
#pragma unroll
      for (int kk = 0; kk < 8; ++kk) a[kk] = make_float2(0.f, 0.f);
      int k = k_lo;
      for (; k + 8 <= k_hi; k += 8) {
        float2 v[8];
#pragma unroll
        for (int kk = 0; kk < 8; ++kk)
          v[kk] = ok ? *reinterpret_cast<const float2*>(part + ((int64_t)(k + kk) * 2 + 0) * D + jc) : make_float2(0.f, 0.f);
#pragma unroll
        for (int kk = 0; kk < 8; ++kk) {
          a[kk].x += v[kk].x;
          a[kk].y += v[kk].y;
        }
      }
      for (; k < k_hi; ++k) {
        const float2 v = ok ? *reinterpret_cast<const float2*>(part + ((int64_t)k * 2 + 0) * D + jc) : make_float2(0.f, 0.f);
        a[0].x += v.x;
        a[0].y += v.y;
      }
      red[w][jc & 255] = ((a[0].x + a[1].x) + (a[2].x + a[3].x)) + ((a[4].x + a[5].x) + (a[6].x + a[7].x));
      red[w][(jc + 1) & 255] = ((a[0].y + a[1].y) + (a[2].y + a[3].y)) + ((a[4].y + a[5].y) + (a[6].y + a[7].y));
      __syncthreads();
      if (w == 0) {
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          const int j = 64 * q + lane;
          if (j < D) {
            float acc = part[((int64_t)c0 * 2 + 1) * D + j];
            for (int v = 0; v < FIX_WAVES; ++v) acc += red[v][j];
            dE[(int64_t)u * D + j] = acc;
          }
        }
      }
      __syncthreads();
      continue;
    }
    for (int j0 = 0; j0 < D; j0 += 256) {
      bool ok[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) ok[q] = j0 + q * 64 + lane < D;
      float a[4][4] = {};  // [column group][accumulator]
      int k = k_lo;
      for (; k + 4 <= k_hi; k += 4)
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
          const float* pr = part + ((int64_t)(k + kk) * 2 + 0) * D + j0 + lane;
#pragma unroll
          for (int q = 0; q < 4; ++q)
            if (ok[q]) a[q][kk] += pr[q * 64];
        }
      for (; k < k_hi; ++k) {
        const float* pr = part + ((int64_t)k * 2 + 0) * D + j0 + lane;
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (ok[q]) a[q][0] += pr[q * 64];
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) red[w][q * 64 + lane] = (a[q][0] + a[q][1]) + (a[q][2] + a[q][3]);
      __syncthreads();
      if (w == 0) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int j = j0 + q * 64 + lane;
          if (j < D) {
            float acc = part[((int64_t)c0 * 2 + 1) * D + j];
            for (int v = 0; v < FIX_WAVES; ++v) acc += red[v][q * 64 + lane];
            dE[(int64_t)u * D + j] = acc;
          }
        }
      }
      __syncthreads();
    }
  }
}

// ---------------------------------------------------------------------------
// generic backward (any shape; plain VALU).  A block claims a chunk: up to 32
// consecutive slices of one (t, i2) run, so every slice of it has the same
// B = G2[t][i2], which is staged in LDS once per chunk (rows padded by one float,
// so reads across a's take distinct banks) when it fits.  Per slice: A staged; C
// recomputed (or reloaded from the checkpoint); the slice's rows in batches whose
// dE rows are staged together: dD per row into dG3, the rows' dC summed; then dA
// into the slice's partial and dB = A^T (sum dC) summed over the chunk (in LDS
// when it fits, else in the chunk's partial in global memory, each element owned
// by one thread) into the chunk's partial; dD of every row into the row's partial.
// No two blocks write one partial, and the fixed-order segment sums below turn the
// partials into dG1 (over the slices of (t, i1)), dG2 (over the chunks of
// (t, i2)) and dG3 (over the rows of (t, i3)).
// ---------------------------------------------------------------------------
constexpr int BWD_LDS_FLOATS = 40448;  // dynamic LDS budget (158 KB of the 160 KB)
constexpr int BWD_DE_FLOATS = 4096;    // dE rows staged per batch

// o = q * div + r along o = o0, o0 + step, ...: the quotient and remainder kept by
// increments (one division at the start, none per step)
struct StepQR {
  int q, r, dq, dr, div;
  __device__ __forceinline__ StepQR(int o0, int step, int d) : div(d) {
    q = o0 / d;
    r = o0 - q * d;
    dq = step / d;
    dr = step - dq * d;
  }
  __device__ __forceinline__ void next() {
    q += dq;
    r += dr;
    if (r >= div) {
      r -= div;
      ++q;
    }
  }
};

// sum over k < n of x[k * xs] * y[k * ys], four independent partial sums
__device__ __forceinline__ float dot_strided(const float* x, int xs, const float* y, int ys, int n) {
  float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
  int k = 0;
  for (; k + 4 <= n; k += 4) {
    a0 = fmaf(x[k * xs], y[k * ys], a0);
    a1 = fmaf(x[(k + 1) * xs], y[(k + 1) * ys], a1);
    a2 = fmaf(x[(k + 2) * xs], y[(k + 2) * ys], a2);
    a3 = fmaf(x[(k + 3) * xs], y[(k + 3) * ys], a3);
  }
  for (; k < n; ++k) a0 = fmaf(x[k * xs], y[k * ys], a0);
  return (a0 + a1) + (a2 + a3);
}

struct GenericBwdPlan {
  int stage_b;  // B in LDS
  int db_lds;   // dB summed over the chunk in LDS
  int rows;     // dE rows per batch
  size_t lds_floats;
};

static GenericBwdPlan generic_bwd_plan(const Shape& s) {
  GenericBwdPlan pl;
  const size_t nC = (size_t)s.d1 * s.d2 * s.R, nB = (size_t)s.R * s.d2 * s.R;
  const size_t bs = (size_t)s.R * (s.d2 * s.R + 1);
  int rows = BWD_DE_FLOATS / s.D;
  rows = rows < 1 ? 1 : (rows > SLICE_ROWS ? SLICE_ROWS : rows);
  pl.rows = rows;
  const size_t base = 2 * nC + (size_t)s.d1 * s.R + (size_t)rows * s.D;
  pl.stage_b = base + bs <= (size_t)BWD_LDS_FLOATS;
  pl.db_lds = base + (pl.stage_b ? bs : 0) + nB <= (size_t)BWD_LDS_FLOATS;
  pl.lds_floats = base + (pl.stage_b ? bs : 0) + (pl.db_lds ? nB : 0);
  return pl;
}

// BWD_THREADS = 1024 (sixteen waves: at a block per CU, four per SIMD hide latency)
// for large products, 256 for small ones (where a block's barriers dominate)
template <int BWD_THREADS>
__global__ void __launch_bounds__(BWD_THREADS) k_bwd_generic(ShapeArgs s, const float* __restrict__ G1,
                                                             const float* __restrict__ G2,
                                                             const float* __restrict__ G3,
                                                             const int4* __restrict__ slices,
                                                             const int4* __restrict__ chunks,
                                                             const uint32_t* __restrict__ run_base,
                                                             const int32_t* __restrict__ uniq_i3,
                                                             int32_t* __restrict__ ctr, const float* __restrict__ dE,
                                                             float* __restrict__ dApart, float* __restrict__ dBpart,
                                                             float* __restrict__ dDpart, float* __restrict__ ckpt,
                                                             int32_t* __restrict__ ckpt_tag, int stage_b, int db_lds,
                                                             int rows_per_batch) {
  extern __shared__ float lds[];
  const int d2R = s.d2 * s.R;
  const int nC = s.d1 * d2R;
  const int nB = s.R * d2R;
  const int bp = stage_b ? d2R + 1 : d2R;  // row pitch of B as read below
  float* C = lds;                          // nC
  float* dCs = C + nC;                     // nC: sum of dC over the slice's rows
  float* As = dCs + nC;                    // d1 * R
  float* dEb = As + s.d1 * s.R;            // rows_per_batch * D
  float* Bs = dEb + rows_per_batch * s.D;  // R * (d2R + 1) when stage_b
  float* dBs = Bs + (stage_b ? s.R * bp : 0);  // nB when db_lds
  __shared__ int s_chunk, s_flag;
  const int nsl = ctr[C_NSLICES];
  const int nchunks = (int)run_base[s.T * s.n2];
  int victim = 0;
  int next = share_lo(nchunks, (int)gridDim.x, (int)blockIdx.x);
  int cur_pg = -1;
  const int rows12 = s.d1 * s.d2;
  // lanes per dC output: 4, 2 or 1, so that the phase keeps the block's threads busy
  const int g_dc = nC * 4 <= BWD_THREADS ? 4 : (nC * 2 <= BWD_THREADS ? 2 : 1);
  const int g_dc_shift = g_dc == 4 ? 2 : (g_dc == 2 ? 1 : 0);
  // dD tasks: each of the R d3 elements taken by g_dd threads (over every g_dd-th row)
  const int RD = s.R * s.d3;
  const int g_dd = RD >= BWD_THREADS ? 1 : (BWD_THREADS / RD < SLICE_ROWS ? BWD_THREADS / RD : SLICE_ROWS);
  while (true) {
    const int c = claim_block_sched(s.sched, ctr + C_BWD_CTR, nchunks, blockIdx.x % SCHED_NQ, &victim, &s_chunk,
                                    &next);
    if (c < 0) break;
    const int4 ch = chunks[c];
    const int s0 = ch.x, s1 = ch.x + ch.y;
    const int run = ch.z;  // t * n2 + i2
    const int t = run / s.n2;
    const float* Bg = G2 + (int64_t)run * nB;
    float* g2 = dBpart + (int64_t)c * nB;  // this chunk's dB partial
    __syncthreads();  // the previous chunk is done with Bs and dBs
    if (stage_b) {
      StepQR ix(threadIdx.x, BWD_THREADS, d2R);
      for (int o = threadIdx.x; o < nB; o += BWD_THREADS, ix.next()) Bs[ix.q * bp + ix.r] = Bg[o];
    }
    const float* Bm = stage_b ? Bs : Bg;
    if (db_lds)
      for (int o = threadIdx.x; o < nB; o += BWD_THREADS) dBs[o] = 0.f;
    for (int si = s0; si < s1; ++si) {
      const int4 sl = slices[si];
      const int p = sl.x, rb = sl.y, re = sl.z;
      const int i1 = (int)(((uint32_t)sl.w % (uint32_t)s.n12) / (uint32_t)s.n2);
      const float* Ag = G1 + ((int64_t)(t * s.n1 + i1) * s.d1) * s.R;
      __syncthreads();  // the previous slice is done with As, C and dCs
      for (int o = threadIdx.x; o < s.d1 * s.R; o += BWD_THREADS) As[o] = Ag[o];
      for (int o = threadIdx.x; o < nC; o += BWD_THREADS) dCs[o] = 0.f;
      __syncthreads();
      if (p != cur_pg) {
        // C recomputed, or with the checkpoint reloaded / published as in the forward
        const bool ck = s.sched == SCHED_STEAL_CKPT;
        if (!(ck && ckpt_load(ckpt, ckpt_tag, p, C, nC, &s_flag))) {
          StepQR ix(threadIdx.x, BWD_THREADS, d2R);  // (j1, column)
          for (int o = threadIdx.x; o < nC; o += BWD_THREADS, ix.next())
            C[o] = dot_strided(As + ix.q * s.R, 1, Bm + ix.r, bp, s.R);
          if (ck && s1 < nsl && slices[s1].x == p) {  // the group goes on past this chunk
            __syncthreads();
            ckpt_store(ckpt, ckpt_tag, p, C, nC, &s_flag);
          }
        }
        cur_pg = p;
        __syncthreads();
      }
      for (int u0 = rb; u0 < re; u0 += rows_per_batch) {
        const int nr = re - u0 < rows_per_batch ? re - u0 : rows_per_batch;
        for (int o = threadIdx.x; o < nr * s.D; o += BWD_THREADS) dEb[o] = dE[(int64_t)u0 * s.D + o];
        __syncthreads();
        // dD_u = C^T dE_u  (R x d3) per row: task (part, e) takes element e = (b, j3) of
        // rows part, part + g_dd, ... of the batch
        for (int tk = threadIdx.x; tk < g_dd * RD; tk += BWD_THREADS) {
          const int part = tk / RD, e = tk - part * RD;
          const int b = e / s.d3, j3 = e - b * s.d3;
          for (int rr = part; rr < nr; rr += g_dd) {
            dDpart[(int64_t)(u0 + rr) * RD + e] = dot_strided(C + b, s.R, dEb + rr * s.D + j3, s.d3, rows12);
          }
        }
        // dC = sum over the batch's rows of dE_u D_u^T; with fewer outputs than threads,
        // g consecutive lanes share an output (each every g-th row), combined by shuffles
        StepQR dcx((int)threadIdx.x >> g_dc_shift, BWD_THREADS >> g_dc_shift, s.R);  // (r, b) of o
        for (int base = 0; base < g_dc * nC; base += BWD_THREADS, dcx.next()) {
          const int og = base + (int)threadIdx.x;
          const bool ok = og < g_dc * nC;
          const int o = og >> g_dc_shift, part = og & (g_dc - 1);
          const int r = dcx.q, b = dcx.r;
          float acc = 0.f;
          if (ok)
            for (int rr = part; rr < nr; rr += g_dc) {
              const int i3 = uniq_i3[u0 + rr];
              const float* Dm = G3 + ((int64_t)(t * s.n3 + i3) * s.R + b) * s.d3;
              const float* de = dEb + rr * s.D + r * s.d3;
              for (int j3 = 0; j3 < s.d3; ++j3) acc = fmaf(de[j3], Dm[j3], acc);
            }
          if (g_dc >= 2) acc += __shfl_xor(acc, 1, 64);
          if (g_dc >= 4) acc += __shfl_xor(acc, 2, 64);
          if (ok && part == 0) dCs[o] += acc;
        }
        __syncthreads();
      }
      // dA = (sum dC) B^T  (d1 x R), dB = A^T (sum dC)  (R x d2R)
      // dA: four consecutive lanes per output, each over every fourth term, combined by
      // shuffles within the wave (the loop runs whole block strides so every lane takes
      // part in the shuffles)
      float* g1 = dApart + (int64_t)si * s.d1 * s.R;  // this slice's dA partial
      StepQR dax((int)threadIdx.x >> 2, BWD_THREADS >> 2, s.R);  // (j1, a) of o
      for (int base = 0; base < 4 * s.d1 * s.R; base += BWD_THREADS, dax.next()) {
        const int o4 = base + (int)threadIdx.x;
        const bool ok = o4 < 4 * s.d1 * s.R;
        const int o = o4 >> 2, part = o4 & 3;
        const int j1 = ok ? dax.q : 0, a = ok ? dax.r : 0;
        const int nterm = d2R > part ? (d2R - part + 3) >> 2 : 0;
        float v = ok ? dot_strided(dCs + j1 * d2R + part, 4, Bm + a * bp + part, 4, nterm) : 0.f;
        v += __shfl_xor(v, 1, 64);
        v += __shfl_xor(v, 2, 64);
        if (ok && part == 0) g1[o] = v;
      }
      StepQR dbx(threadIdx.x, BWD_THREADS, d2R);  // (a, column)
      for (int o = threadIdx.x; o < nB; o += BWD_THREADS, dbx.next()) {
        const int a = dbx.q, cc = dbx.r;
        float acc = 0.f;
        for (int j1 = 0; j1 < s.d1; ++j1) acc = fmaf(As[j1 * s.R + a], dCs[j1 * d2R + cc], acc);
        // each thread owns its elements across the chunk's slices
        if (db_lds)
          dBs[o] += acc;
        else
          g2[o] = si == s0 ? acc : g2[o] + acc;
      }
    }
    if (db_lds)
      for (int o = threadIdx.x; o < nB; o += BWD_THREADS) g2[o] = dBs[o];
  }
}

// ---------------------------------------------------------------------------
// Fixed-order segment sums of the generic backward's partials.  Each writes its
// sum into the gradient, or with update set subtracts lr times it from the core
// itself (the fused backward-and-SGD call; the fused kernel has finished reading
// the cores).  Every element of its core is visited exactly once; untouched
// slices get zero (or are left as they are by the update).
// ---------------------------------------------------------------------------
constexpr int GRED_THREADS = 256;

__device__ __forceinline__ void put_g(float* out, int64_t i, float acc, float lr, bool update) {
  out[i] = update ? out[i] - lr * acc : acc;
}

// Eight accumulators take consecutive terms of an ordered list in turn (eight loads
// in flight per thread); their fixed tree sum is the segment's sum.
__device__ __forceinline__ float sum8(const float (&a)[8]) {
  return ((a[0] + a[1]) + (a[2] + a[3])) + ((a[4] + a[5]) + (a[6] + a[7]));
}

// dG1[t][i1] = sum of the dA partials of the slices of prefixes (i1, i2), i2 ascending
// (each prefix's slices in order); block (t i1, column block).  Each round of
// GRED_THREADS prefixes is scanned into a list of slice ids in LDS (G1_WIN at a
// time), which every column then walks in list order.
constexpr int G1_WIN = 2048;
__global__ void __launch_bounds__(GRED_THREADS) k_gred_g1(ShapeArgs s, const uint32_t* __restrict__ dense_cnt,
                                                          const uint32_t* __restrict__ dense_base,
                                                          const float* __restrict__ dApart, float* __restrict__ dG1,
                                                          float lr, bool update) {
  __shared__ uint32_t wsum[GRED_THREADS / 64];
  __shared__ uint32_t list[G1_WIN];
  const int ti1 = blockIdx.x;
  const int t = ti1 / s.n1, i1 = ti1 - t * s.n1;
  const int d1R = s.d1 * s.R;
  const int e = blockIdx.y * GRED_THREADS + threadIdx.x;
  const bool col = e < d1R;
  float a[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int r0 = 0; r0 < s.n2; r0 += GRED_THREADS) {
    const int i2 = r0 + (int)threadIdx.x;
    uint32_t cnt = 0, base = 0;
    if (i2 < s.n2) {
      const int64_t slot = ((int64_t)t * s.n2 + i2) * s.n1 + i1;
      cnt = dense_cnt[slot];
      base = dense_base[slot];
    }
    uint32_t total;
    const uint32_t pos = block_excl_scan<uint32_t, GRED_THREADS>(cnt, wsum, &total);
    for (uint32_t w0 = 0; w0 < total; w0 += G1_WIN) {
      const uint32_t k0 = pos > w0 ? pos : w0;
      const uint32_t k1 = pos + cnt < w0 + G1_WIN ? pos + cnt : w0 + G1_WIN;
      for (uint32_t k = k0; k < k1; ++k) list[k - w0] = base + (k - pos);
      __syncthreads();
      const int wn = (int)(total - w0 < (uint32_t)G1_WIN ? total - w0 : (uint32_t)G1_WIN);
      if (col) {
        int j = 0;
        for (; j + 8 <= wn; j += 8) {
          float v[8];
#pragma unroll
          for (int q = 0; q < 8; ++q) v[q] = ntl(dApart + (int64_t)list[j + q] * d1R + e);
#pragma unroll
          for (int q = 0; q < 8; ++q) a[q] += v[q];
        }
        for (; j < wn; ++j) a[0] += ntl(dApart + (int64_t)list[j] * d1R + e);
      }
      __syncthreads();  // the list is refilled
    }
  }
  if (col) put_g(dG1, (int64_t)ti1 * d1R + e, sum8(a), lr, update);
}

// dG2[t][i2] = sum of the dB partials of the chunks of run (t, i2), in chunk order
__global__ void __launch_bounds__(GRED_THREADS) k_gred_g2(const uint32_t* __restrict__ run_base,
                                                          const float* __restrict__ dBpart, int nB,
                                                          float* __restrict__ dG2, float lr, bool update) {
  const int r = blockIdx.x;
  const int e = blockIdx.y * GRED_THREADS + threadIdx.x;
  if (e >= nB) return;
  const int c0 = (int)run_base[r], c1 = (int)run_base[r + 1];
  float a[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  int c = c0;
  for (; c + 8 <= c1; c += 8) {
    float v[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) v[q] = dBpart[(int64_t)(c + q) * nB + e];
#pragma unroll
    for (int q = 0; q < 8; ++q) a[q] += v[q];
  }
  for (; c < c1; ++c) a[0] += dBpart[(int64_t)c * nB + e];
  put_g(dG2, (int64_t)r * nB + e, sum8(a), lr, update);
}

// Sort keys t n3 + i3 of the unique rows (positions from U on get `sentinel`, which
// sorts last), values = row ids
__global__ void k_g3_keys(ShapeArgs s, const uint32_t* __restrict__ uniq_key, const int32_t* __restrict__ ctr, int n,
                          uint32_t sentinel, uint32_t* __restrict__ keys, uint32_t* __restrict__ vals) {
  const int U = ctr[C_U];
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) {
    uint32_t k = sentinel;
    if (i < U) {
      const Digits d = decode_key(uniq_key[i], s.Npad, s.n2, s.n3);
      k = (uint32_t)d.t * (uint32_t)s.n3 + (uint32_t)d.i3;
    }
    keys[i] = k;
    vals[i] = (uint32_t)i;
  }
}

// [lo, hi) of every (t, i3) in the sorted rows (bins no row falls in keep lo = hi = 0)
__global__ void k_g3_bins(const uint32_t* __restrict__ keys, const int32_t* __restrict__ ctr, int32_t* __restrict__ lo,
                          int32_t* __restrict__ hi) {
  const int U = ctr[C_U];
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < U; i += gridDim.x * blockDim.x) {
    const uint32_t k = keys[i];
    if (i == 0 || keys[i - 1] != k) lo[k] = i;
    if (i == U - 1 || keys[i + 1] != k) hi[k] = i + 1;
  }
}

// dG3[t][i3] = sum of the dD partials of the rows of (t, i3), in row order
__global__ void __launch_bounds__(GRED_THREADS) k_gred_g3(const int32_t* __restrict__ lo,
                                                          const int32_t* __restrict__ hi,
                                                          const uint32_t* __restrict__ rows,
                                                          const float* __restrict__ dDpart, int RD,
                                                          float* __restrict__ dG3, float lr, bool update) {
  const int b = blockIdx.x;
  const int e = blockIdx.y * GRED_THREADS + threadIdx.x;
  if (e >= RD) return;
  const int k0 = lo[b], k1 = hi[b];
  float a[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  int k = k0;
  for (; k + 8 <= k1; k += 8) {
    float v[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) v[q] = ntl(dDpart + (int64_t)rows[k + q] * RD + e);
#pragma unroll
    for (int q = 0; q < 8; ++q) a[q] += v[q];
  }
  for (; k < k1; ++k) a[0] += ntl(dDpart + (int64_t)rows[k] * RD + e);
  put_g(dG3, (int64_t)b * RD + e, sum8(a), lr, update);
}

static int bits_of(uint64_t x) {
  int b = 0;
  while (x) {
    ++b;
    x >>= 1;
  }
  return b;
}

// The three segment sums of the generic backward (M sorted occurrences bound the rows).
// The segment sums of the generic and R = 64 paths.  After the R = 64 MFMA backward
// (dg2_from_dc), dG2 comes from the per-slice dC partials by a product with G1, which
// runs before the dG1 sums: with `update` those overwrite G1.
static hipError_t launch_generic_reduce(const Shape& s, const Work& w, int64_t M, const float* G1, float* dG1,
                                        float* dG2, float* dG3, float lr, bool update, bool dg2_from_dc,
                                        hipStream_t st) {
  const int d1R = s.d1 * s.R, nB = s.R * s.d2 * s.R, RD = s.R * s.d3;
  const int n = (int)M;
  const uint32_t nbins = (uint32_t)s.T * (uint32_t)s.n3;
  hipLaunchKernelGGL(k_g3_keys, dim3((n + 255) / 256 < 4096 ? (n + 255) / 256 : 4096), dim3(256), 0, st,
                     shape_args(s), (const uint32_t*)w.uniq_key, (const int32_t*)w.ctr, n, nbins, w.g3keys[0],
                     w.g3vals[0]);
  int res = 0;
  hipError_t e = sort_pairs(w, w.g3keys, w.g3vals, n, bits_of(nbins), &res, st);
  if (e != hipSuccess) return e;
  if ((e = fill_u32(reinterpret_cast<uint32_t*>(w.g3lo), nbins, 0u, st)) != hipSuccess) return e;
  if ((e = fill_u32(reinterpret_cast<uint32_t*>(w.g3hi), nbins, 0u, st)) != hipSuccess) return e;
  hipLaunchKernelGGL(k_g3_bins, dim3((n + 255) / 256 < 4096 ? (n + 255) / 256 : 4096), dim3(256), 0, st,
                     (const uint32_t*)w.g3keys[res], (const int32_t*)w.ctr, w.g3lo, w.g3hi);
  hipLaunchKernelGGL(k_gred_g3, dim3(nbins, (RD + GRED_THREADS - 1) / GRED_THREADS), dim3(GRED_THREADS), 0, st,
                     (const int32_t*)w.g3lo, (const int32_t*)w.g3hi, (const uint32_t*)w.g3vals[res],
                     (const float*)w.dDpart, RD, dG3, lr, update);
  if (dg2_from_dc && (e = launch_dg2_r64(s, w, G1, dG2, lr, update, st)) != hipSuccess) return e;
  hipLaunchKernelGGL(k_gred_g1, dim3(s.T * s.n1, (d1R + GRED_THREADS - 1) / GRED_THREADS), dim3(GRED_THREADS), 0, st,
                     shape_args(s), (const uint32_t*)w.dense_cnt, (const uint32_t*)w.dense_base,
                     (const float*)w.dApart, dG1, lr, update);
  if (!dg2_from_dc)
    hipLaunchKernelGGL(k_gred_g2, dim3(s.T * s.n2, (nB + GRED_THREADS - 1) / GRED_THREADS), dim3(GRED_THREADS), 0,
                       st, (const uint32_t*)w.run_nch, (const float*)w.dBpart, nB, dG2, lr, update);
  return hipGetLastError();
}

hipError_t launch_backward(const Shape& s, const Work& w, const float* G1, const float* G2, const float* G3,
                           const int64_t* offsets, int64_t M, int64_t B, const float* dV, float* dG1, float* dG2,
                           float* dG3, float lr, bool update, const Prof& prof, hipStream_t st) {
  (void)offsets;
  (void)B;
  hipError_t e;
  const bool fast = bwd_r32_supported(s, w.M);
  // With update set, dG1..dG3 are the cores themselves: both paths apply the update
  // in their final segment sums, after the fused kernel has read the cores.
  if (M <= 0) {
    if (update) return hipSuccess;  // zero gradients: the update leaves the cores as they are
    const int64_t n1s = (int64_t)s.T * s.n1 * s.d1 * s.R;
    const int64_t n2s = (int64_t)s.T * s.n2 * s.R * s.d2 * s.R;
    const int64_t n3s = (int64_t)s.T * s.n3 * s.R * s.d3;
    if ((e = fill_f32(dG1, n1s, 0.f, st)) != hipSuccess) return e;
    if ((e = fill_f32(dG2, n2s, 0.f, st)) != hipSuccess) return e;
    return fill_f32(dG3, n3s, 0.f, st);
  }
  float* dE = w.E;
  const int nseg = (int)((M + SEG_CHUNK - 1) / SEG_CHUNK);
  hipLaunchKernelGGL(k_sorted_bag, dim3(xcd_grid((unsigned)((M + SB_ITEMS * 256 - 1) / (SB_ITEMS * 256)))), dim3(256),
                     0, st, (const uint32_t*)w.sorted_pos, (const int32_t*)w.bag_of, (const int32_t*)w.ctr,
                     w.sorted_bag);
  prof_begin(prof, K_SEG_SUM, st);
  if (s.D == 128 || s.D == 32) {
    hipLaunchKernelGGL(s.D == 128 ? k_seg_dE128 : k_seg_dE32, dim3(xcd_grid((nseg + SEG_WAVES - 1) / SEG_WAVES)),
                       dim3(64 * SEG_WAVES), 0, st, dV, (const int32_t*)w.sorted_uid, (const int32_t*)w.sorted_bag,
                       (const int32_t*)w.occ_start, (const int32_t*)w.ctr, dE, w.seg_part);
  } else {
    hipLaunchKernelGGL(k_seg_dE, dim3((nseg + SEG_WAVES - 1) / SEG_WAVES), dim3(64 * SEG_WAVES), 0, st, dV, (const int32_t*)w.sorted_uid,
                       (const int32_t*)w.sorted_bag, (const int32_t*)w.occ_start,
                       (const int32_t*)w.ctr, s.D, dE, w.seg_part);
  }
  prof_end(prof, K_SEG_SUM, st);
  hipLaunchKernelGGL(k_seg_fix, dim3((nseg + FIX_SCREEN - 1) / FIX_SCREEN), dim3(64 * FIX_WAVES), 0, st, (const int32_t*)w.sorted_uid, (const int32_t*)w.occ_start,
                     (const int32_t*)w.ctr, s.D, (const float*)w.seg_part, dE);
  if (fast) return launch_bwd_r32(s, w, G1, G2, G3, dG1, dG2, dG3, lr, update, prof, st);
  if (!w.dDpart || !w.g3lo) return hipErrorInvalidValue;
  if (bwd_r64_supported(s, w.M)) {  // MFMA partials, then the same segment sums (dG2 by a product)
    if (!w.dCpart) return hipErrorInvalidValue;
    if ((e = launch_bwd_r64(s, w, G1, G2, G3, prof, st)) != hipSuccess) return e;
    return launch_generic_reduce(s, w, M, G1, dG1, dG2, dG3, lr, update, true, st);
  }
  const int grid = persistent_grid() * 2;
  if ((e = fill_u32(reinterpret_cast<uint32_t*>(w.ctr + C_BWD_CTR), SCHED_NQ * SCHED_STRIDE, 0u, st)) != hipSuccess)
    return e;
  const GenericBwdPlan pl = generic_bwd_plan(s);
  const size_t lds = sizeof(float) * pl.lds_floats;
  const bool wide = (int64_t)s.d1 * s.d2 * s.R >= 1024 || s.D >= 128;
  const void* kfn = wide ? (const void*)k_bwd_generic<1024> : (const void*)k_bwd_generic<256>;
  if ((e = hipFuncSetAttribute(kfn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds)) != hipSuccess) return e;
  if (s.sched == SCHED_STEAL_CKPT) {  // the forward's checkpoints may hold other cores' C
    if (!w.ckpt_tag) return hipErrorInvalidValue;
    if ((e = fill_u32(reinterpret_cast<uint32_t*>(w.ckpt_tag), CKPT_SLOTS, (uint32_t)CKPT_EMPTY, st)) != hipSuccess)
      return e;
  }
  prof_begin(prof, K_BWD_FUSED, st);
  if (wide)
    hipLaunchKernelGGL(k_bwd_generic<1024>, dim3(grid), dim3(1024), lds, st, shape_args(s), G1, G2, G3,
                       (const int4*)w.slices, (const int4*)w.chunks, (const uint32_t*)w.run_nch,
                       (const int32_t*)w.uniq_i3, w.ctr, (const float*)dE, w.dApart, w.dBpart, w.dDpart, w.ckpt,
                       w.ckpt_tag, pl.stage_b, pl.db_lds, pl.rows);
  else
    hipLaunchKernelGGL(k_bwd_generic<256>, dim3(grid), dim3(256), lds, st, shape_args(s), G1, G2, G3,
                       (const int4*)w.slices, (const int4*)w.chunks, (const uint32_t*)w.run_nch,
                       (const int32_t*)w.uniq_i3, w.ctr, (const float*)dE, w.dApart, w.dBpart, w.dDpart, w.ckpt,
                       w.ckpt_tag, pl.stage_b, pl.db_lds, pl.rows);
  prof_end(prof, K_BWD_FUSED, st);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  return launch_generic_reduce(s, w, M, G1, dG1, dG2, dG3, lr, update, false, st);
}

// ---------------------------------------------------------------------------
// SGD: G -= lr * dG on the three cores
// ---------------------------------------------------------------------------
__global__ void k_sgd(float* __restrict__ G, const float* __restrict__ dG, int64_t n, float lr) {
  int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int64_t n4 = n / 4;
  float4* G4 = reinterpret_cast<float4*>(G);
  const float4* d4 = reinterpret_cast<const float4*>(dG);
  for (int64_t k = i; k < n4; k += stride) {
    float4 g = G4[k], d = d4[k];
    g.x = fmaf(-lr, d.x, g.x);
    g.y = fmaf(-lr, d.y, g.y);
    g.z = fmaf(-lr, d.z, g.z);
    g.w = fmaf(-lr, d.w, g.w);
    G4[k] = g;
  }
  for (int64_t k = n4 * 4 + i; k < n; k += stride) G[k] = fmaf(-lr, dG[k], G[k]);
}

hipError_t launch_sgd(const Shape& s, float* G1, float* G2, float* G3, const float* dG1, const float* dG2,
                      const float* dG3, float lr, hipStream_t st) {
  const int64_t n[3] = {(int64_t)s.T * s.n1 * s.d1 * s.R, (int64_t)s.T * s.n2 * s.R * s.d2 * s.R,
                        (int64_t)s.T * s.n3 * s.R * s.d3};
  float* G[3] = {G1, G2, G3};
  const float* d[3] = {dG1, dG2, dG3};
  for (int k = 0; k < 3; ++k) {
    hipError_t e = launch_sgd1(G[k], d[k], n[k], lr, st);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_sgd1(float* G, const float* dG, int64_t n, float lr, hipStream_t st) {
  int64_t blocks = (n / 4 + 255) / 256;
  if (blocks < 1) blocks = 1;
  if (blocks > 2048) blocks = 2048;
  hipLaunchKernelGGL(k_sgd, dim3((unsigned)blocks), dim3(256), 0, st, G, dG, n, lr);
  return hipGetLastError();
}

}  // namespace ttemb
